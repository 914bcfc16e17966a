// Gated delta-rule write of the visual tokens into a linear-attention (Gated DeltaNet) state
// (appendix on linear attention, Eq. 15-16), per sequence b and value head h:
//     S <- alpha_t S;   S <- S + beta_t k_t (v_t - S^T k_t)^T         t = 0 .. N-1.
//
// Chunked form (chunks of C = 64 tokens). Inside a chunk, with g_t = sum_{s<=t} log alpha_s,
// gamma_t = exp(g_t) and the chunk's initial state S_0, every step adds a rank-one term, so
//     S_t = gamma_t S_0 + sum_{s<=t} (gamma_t / gamma_s) k_s u_s^T,
// and the pseudo-values u solve the unit lower-triangular system
//     (I + A) U = diag(beta) (V - diag(gamma) K S_0),   A[t][s] = beta_t (gamma_t/gamma_s) k_t.k_s, s < t.
// With T = (I + A)^-1, U = Uv - W S_0 where Uv = T diag(beta) V and W = T diag(beta gamma) K do
// not depend on the state, and the state after the chunk is
//     S_C = gamma_C S_0 + Kt U,   Kt = (diag(gamma_C / gamma) K)^T.
// k_gdr_prep computes Uv, W, Kt and gamma_C for every chunk in parallel (MFMA for K K^T and
// the two products, fp32 forward substitution for T); k_gdr_scan then runs the chunks in
// order, U = Uv - W S and S = gamma_C S + Kt U, with the fp32 state in MFMA accumulators. The
// rule acts on every state column independently, so the scan splits the value columns over
// workgroups (32 per block). Products read the state rounded to the call dtype; the state
// itself stays fp32.
#include "delta_rule.hpp"

#include <algorithm>
#include <cfloat>
#include <cmath>

#include "dv_device.hpp"

namespace dv {

namespace gdr {
constexpr int C = 64;     // tokens per chunk
constexpr int PAD = 8;    // elements of padding per LDS row (bank spread)
constexpr int NT = 256;   // threads per block (4 waves)
}  // namespace gdr

template <typename T>
__device__ __forceinline__ typename Frag8<T>::type frag_load(const T* p) {
  typedef typename Frag8<T>::type F;
  return *(const F*)p;
}

template <typename T>
__device__ __forceinline__ typename Frag8<T>::type frag_zero() {
  return typename Frag8<T>::type{};
}

// LDS layout of k_gdr_prep (byte offsets). For bf16, T diag(beta) and T diag(beta gamma)
// (unpadded rows) reuse the bytes of A, which is dead once A21 T11 is formed; the block then
// stays under 80 KiB so that two share a CU.
template <typename T, int DK, int DV>
struct GdrLds {
  static constexpr int C = gdr::C, P = gdr::PAD;
  static constexpr bool kReuse = sizeof(T) == 2;
  static constexpr int TWP = kReuse ? C : C + P;                          // pitch of Tu, Tw
  static constexpr size_t g = 0;                                          // float[C]  g_t
  static constexpr size_t beta = g + C * 4;                               // float[C]
  static constexpr size_t am = beta + C * 4;                              // float[C][C]  A
  static constexpr size_t tf = am + (size_t)C * C * 4;                    // float[C][C+1] T (fp32)
  static constexpr size_t xb = tf + (size_t)C * (C + 1) * 4;              // float[32][33] A21 T11
  static constexpr size_t vt = xb + (size_t)32 * 33 * 4;                  // T[DV][C+P] V^T
  static constexpr size_t kt = vt + (size_t)DV * (C + P) * sizeof(T);     // T[DK][C+P] K^T
  static constexpr size_t end = kt + (size_t)DK * (C + P) * sizeof(T);
  static constexpr size_t tu = kReuse ? am : end;                         // T[C][TWP] T diag(beta)
  static constexpr size_t tw = tu + (size_t)C * TWP * sizeof(T);          // T[C][TWP] T diag(beta gamma)
  static constexpr size_t bytes = kReuse ? end : tw + (size_t)C * TWP * sizeof(T);
  static_assert(!kReuse || 2 * C * TWP * sizeof(T) <= (size_t)C * C * 4, "Tu and Tw fit in A");
};

template <typename T, int DK, int DV>
__global__ __launch_bounds__(gdr::NT) void k_gdr_prep(const T* __restrict__ k,
                                                      const T* __restrict__ v,
                                                      const float* __restrict__ alpha,
                                                      const float* __restrict__ beta, int Hk,
                                                      int Hv, int N, GdrWs ws) {
  using namespace gdr;
  typedef GdrLds<T, DK, DV> L;
  typedef typename Frag8<T>::type F;
  extern __shared__ __align__(16) unsigned char smem[];
  float* g = (float*)(smem + L::g);
  float* bet = (float*)(smem + L::beta);
  float* Am = (float*)(smem + L::am);
  T* Tu = (T*)(smem + L::tu);
  T* Tw = (T*)(smem + L::tw);
  T* VT = (T*)(smem + L::vt);
  T* KT = (T*)(smem + L::kt);
  constexpr int CP = C + PAD;

  const int c = blockIdx.x, hv = blockIdx.y, b = blockIdx.z;
  const int NC = (N + C - 1) / C;
  const int hk = hv / (Hv / Hk);
  const int64_t t0 = (int64_t)c * C;
  const int nval = (int)min((int64_t)C, (int64_t)N - t0);
  const int64_t seq = (int64_t)b * Hv + hv;  // (sequence, value head)
  const T* kc = k + (((int64_t)b * Hk + hk) * N + t0) * DK;
  const T* vc = v + (seq * N + t0) * DV;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int h = lane >> 5, rr = lane & 31;

  // Every global load of the block is issued first, so their latencies overlap: the gates,
  // this thread's pieces of K and V (for the transposed copies) and, for waves 0..2, the
  // fragments of their K K^T tile.
  constexpr int VP = C * (DV / 8) / NT, KP = C * (DK / 8) / NT;  // pieces per thread
  static_assert(C * (DV / 8) % NT == 0 && C * (DK / 8) % NT == 0, "pieces divide the block");
  float la = 0.f, be = 0.f;
  if (wave == 0 && lane < nval) {
    la = alpha[seq * N + t0 + lane];
    be = beta[seq * N + t0 + lane];
  }
  // Piece idx covers token idx % C and channels 8 (idx / C) .. + 7: consecutive lanes take
  // consecutive tokens, so the transposed LDS writes below are contiguous runs.
  F vpc[VP], kpc[KP];
#pragma unroll
  for (int q = 0; q < VP; ++q) {
    const int idx = tid + q * NT, sidx = idx % C, n0 = (idx / C) * 8;
    vpc[q] = sidx < nval ? frag_load<T>(vc + (int64_t)sidx * DV + n0) : frag_zero<T>();
  }
#pragma unroll
  for (int q = 0; q < KP; ++q) {
    const int idx = tid + q * NT, sidx = idx % C, n0 = (idx / C) * 8;
    kpc[q] = sidx < nval ? frag_load<T>(kc + (int64_t)sidx * DK + n0) : frag_zero<T>();
  }
  const int ti3 = wave == 0 ? 0 : 1, si3 = wave == 2 ? 1 : 0;  // K K^T tile of waves 0..2
  F fa3[DK / 16], fb3[DK / 16];
  if (wave < 3) {
    const int ta = ti3 * 32 + rr, sb = si3 * 32 + rr;
#pragma unroll
    for (int ks = 0; ks < DK / 16; ++ks) {
      const int ko = ks * 16 + h * 8;
      fa3[ks] = ta < nval ? frag_load<T>(kc + (int64_t)ta * DK + ko) : frag_zero<T>();
      fb3[ks] = sb < nval ? frag_load<T>(kc + (int64_t)sb * DK + ko) : frag_zero<T>();
    }
  }

  // 1. g_t = prefix sum of log alpha (tokens past N: alpha = 1, beta = 0, k = v = 0).
  if (wave == 0) {
    float x = lane < nval ? __logf(fmaxf(la, FLT_MIN)) : 0.f;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const float y = __shfl_up(x, o, WAVE);
      if (lane >= o) x += y;
    }
    g[lane] = x;
    bet[lane] = be;
  }
  // 2. The chunk's K and V, transposed into LDS (B operands of the two products, and the rows
  //    of Kt).
#pragma unroll
  for (int q = 0; q < VP; ++q) {
    const int idx = tid + q * NT, sidx = idx % C, n0 = (idx / C) * 8;
#pragma unroll
    for (int e = 0; e < 8; ++e) VT[(n0 + e) * CP + sidx] = vpc[q][e];
  }
#pragma unroll
  for (int q = 0; q < KP; ++q) {
    const int idx = tid + q * NT, sidx = idx % C, n0 = (idx / C) * 8;
#pragma unroll
    for (int e = 0; e < 8; ++e) KT[(n0 + e) * CP + sidx] = kpc[q][e];
  }
  __syncthreads();
  const float gC = g[C - 1];

  // 3. A[t][s] = beta_t exp(g_t - g_s) k_t.k_s for s < t (K K^T on MFMA, lower tiles only).
  if (wave < 3) {
    f32x16 acc = {};
#pragma unroll
    for (int ks = 0; ks < DK / 16; ++ks) mfma_k16(acc, fa3[ks], fb3[ks]);
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int t = ti3 * 32 + acc_row(lane, i), sx = si3 * 32 + rr;
      Am[t * C + sx] = sx < t ? bet[t] * __expf(g[t] - g[sx]) * acc[i] : 0.f;
    }
  } else {
    for (int e = lane; e < 32 * 32; e += 64) Am[(e >> 5) * C + 32 + (e & 31)] = 0.f;
  }
  __syncthreads();

  // 4. T = (I + A)^-1 for the unit lower-triangular I + A, as a 2 x 2 block triangle:
  //      T11 = (I + A11)^-1, T22 = (I + A22)^-1, T21 = -T22 A21 T11.
  //    Wave 0 inverts both diagonal blocks by forward substitution (lanes 0..31 the columns
  //    of T11, lanes 32..63 those of T22; each column is zero above its diagonal, so all lanes
  //    run the same unrolled loops with the column in registers and the rows of A read as LDS
  //    broadcasts, summed in four chains). Meanwhile the other waves write
  //    Kt = (diag(gamma_C / gamma) K)^T.
  float* Tf = (float*)(smem + L::tf);
  float* Xb = (float*)(smem + L::xb);
  constexpr int TP = C + 1;
  if (wave == 0) {
    const int half = lane >> 5;            // 0: block (1,1), 1: block (2,2)
    const int j = lane & 31, o = half * 32;
    float col[32];
#pragma unroll
    for (int i = 0; i < 32; ++i) {
      float x4[4] = {0.f, 0.f, 0.f, 0.f};
      const float* arow = Am + (o + i) * C + o;
#pragma unroll
      for (int s4 = 0; s4 < i; s4 += 4) {
        const f32x4 a4 = *(const f32x4*)(arow + s4);
#pragma unroll
        for (int u = 0; u < 4; ++u)
          if (s4 + u < i) x4[u] -= a4[u] * col[s4 + u];
      }
      const float x = (x4[0] + x4[1]) + (x4[2] + x4[3]);
      col[i] = i < j ? 0.f : (i == j ? 1.f : x);
      Tf[(o + i) * TP + o + j] = col[i];
      if (half == 0) Tf[i * TP + 32 + j] = 0.f;  // upper-right block
    }
  } else {
    T* Kt = ws.kt<T>(seq * NC + c, DK);
    for (int idx = tid - 64; idx < DK * (C / 8); idx += NT - 64) {
      const int n = idx / (C / 8), s0 = (idx % (C / 8)) * 8;
      const F x = *(const F*)(KT + n * CP + s0);
      F y;
#pragma unroll
      for (int e = 0; e < 8; ++e) y[e] = from_f32<T>(__expf(gC - g[s0 + e]) * to_f32(x[e]));
      *(F*)(Kt + n * C + s0) = y;
    }
  }
  __syncthreads();
  // X = A21 T11 (32 x 32 x 32), then T21 = -T22 X; four entries per thread.
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int e = tid + q * NT, i = e >> 5, jj = e & 31;
    float x = 0.f;
#pragma unroll 8
    for (int sx = jj; sx < 32; ++sx) x += Am[(32 + i) * C + sx] * Tf[sx * TP + jj];
    Xb[i * 33 + jj] = x;
  }
  __syncthreads();
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const int e = tid + q * NT, i = e >> 5, jj = e & 31;
    float x = 0.f;
#pragma unroll 8
    for (int sx = 0; sx <= i; ++sx) x -= Tf[(32 + i) * TP + 32 + sx] * Xb[sx * 33 + jj];
    Tf[(32 + i) * TP + jj] = x;
  }
  __syncthreads();
  // The products need T diag(beta) and T diag(beta gamma) in the call dtype.
  for (int e = tid; e < C * C; e += NT) {
    const int i = e >> 6, jj = e & 63;
    const float t = Tf[i * TP + jj];
    Tu[i * L::TWP + jj] = from_f32<T>(t * bet[jj]);
    Tw[i * L::TWP + jj] = from_f32<T>(t * bet[jj] * __expf(g[jj]));
  }
  __syncthreads();

  // 5. Uv = (T diag(beta)) V and W = (T diag(beta gamma)) K, 32x32 tiles over the waves.
  constexpr int NU = (C / 32) * (DV / 32), NW = (C / 32) * (DK / 32);
  T* Uv = ws.uv<T>(seq * NC + c, DV);
  T* W = ws.w<T>(seq * NC + c, DK);
  for (int q = wave; q < NU + NW; q += NT / 64) {
    const bool isu = q < NU;
    const int qq = isu ? q : q - NU;
    const int nd = isu ? DV / 32 : DK / 32;
    const int ti = qq / nd, ni = qq % nd;
    const T* As = isu ? Tu : Tw;
    const T* Bs = isu ? VT : KT;
    f32x16 acc = {};
#pragma unroll
    for (int ks = 0; ks < C / 16; ++ks) {
      const int ko = ks * 16 + h * 8;
      mfma_k16(acc, frag_load<T>(As + (ti * 32 + rr) * L::TWP + ko),
               frag_load<T>(Bs + (ni * 32 + rr) * CP + ko));
    }
    T* out = isu ? Uv : W;
    const int ld = isu ? DV : DK;
#pragma unroll
    for (int i = 0; i < 16; ++i)
      out[(ti * 32 + acc_row(lane, i)) * ld + ni * 32 + rr] = from_f32<T>(acc[i]);
  }
  if (tid == 0) ws.gc[seq * NC + c] = __expf(gC);
}

template <typename T, int DK>
struct ScanLds {
  static constexpr int C = gdr::C, P = gdr::PAD;
  static constexpr size_t ssh = 0;                                       // T[32][DK+P]
  static constexpr size_t ush = ssh + (size_t)32 * (DK + P) * sizeof(T);  // T[32][C+P]
  static constexpr size_t bytes = ush + (size_t)32 * (C + P) * sizeof(T);
};

// The chunk step S <- gamma_C S + Kt (Uv - W S) is affine in S, so a run of chunks maps a
// start state S to Phi S + Psi. A long sequence is cut into ws.P segments: k_gdr_scan_seg runs
// every segment at once from the start states I (for Phi, without Uv) and 0 (for Psi), and
// k_gdr_combine_seg then applies the segments in order, S <- Phi_g S + Psi_g. With one segment
// k_gdr_scan reads and writes S directly.
template <typename T, int DK, int DV>
__global__ __launch_bounds__(gdr::NT) void k_gdr_scan(float* __restrict__ S, int Hv, int N,
                                                      GdrWs ws) {
  using namespace gdr;
  typedef typename Frag8<T>::type F;
  typedef ScanLds<T, DK> L;
  extern __shared__ __align__(16) unsigned char smem[];
  T* Ssh = (T*)(smem + L::ssh);  // state slice, [column][dk]: B operand of U = Uv - W S
  T* Ush = (T*)(smem + L::ush);  // U slice, [column][token]: B operand of S += Kt U
  constexpr int SP = DK + PAD, UP = C + PAD;
  const int sl = blockIdx.x * 32, hv = blockIdx.y, b = blockIdx.z;
  const int NC = (N + C - 1) / C;
  const int64_t seq = (int64_t)b * Hv + hv;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int h = lane >> 5, rr = lane & 31;
  const bool holds = wave * 32 < DK;  // this wave keeps state rows [32 wave, 32 wave + 32)
  const bool makes_u = wave * 32 < C;  // this wave computes U rows [32 wave, 32 wave + 32)
  float* Sg = S + seq * DK * DV;

  f32x16 st = {};
  if (holds) {
#pragma unroll
    for (int i = 0; i < 16; ++i) st[i] = Sg[(int64_t)(wave * 32 + acc_row(lane, i)) * DV + sl + rr];
  }
  // Operands of one chunk, loaded one chunk ahead: W rows (A operand of U = Uv - W S), the Uv
  // entries of this lane's accumulator positions, Kt rows (A operand of S += Kt U) and gamma_C.
  F wf[DK / 16], kf[C / 16];
  T uv[16];
  float gcn = 1.f;
  auto fetch = [&](int c) {
    const int64_t cid = seq * NC + c;
    gcn = ws.gc[cid];
    if (makes_u) {
      const T* W = ws.w<T>(cid, DK) + (int64_t)(wave * 32 + rr) * DK;
#pragma unroll
      for (int ks = 0; ks < DK / 16; ++ks) wf[ks] = *(const F*)(W + ks * 16 + h * 8);
      const T* Uv = ws.uv<T>(cid, DV);
#pragma unroll
      for (int i = 0; i < 16; ++i) uv[i] = Uv[(int64_t)(wave * 32 + acc_row(lane, i)) * DV + sl + rr];
    }
    if (holds) {
      const T* Kt = ws.kt<T>(cid, DK) + (int64_t)(wave * 32 + rr) * C;
#pragma unroll
      for (int ks = 0; ks < C / 16; ++ks) kf[ks] = *(const F*)(Kt + ks * 16 + h * 8);
    }
  };
  fetch(0);
  for (int c = 0; c < NC; ++c) {
    F wnow[DK / 16], know[C / 16];
    T unow[16];
#pragma unroll
    for (int q = 0; q < DK / 16; ++q) wnow[q] = wf[q];
#pragma unroll
    for (int q = 0; q < C / 16; ++q) know[q] = kf[q];
#pragma unroll
    for (int q = 0; q < 16; ++q) unow[q] = uv[q];
    const float gc = gcn;
    if (c + 1 < NC) fetch(c + 1);
    // (a) publish the state slice in the call dtype
    if (holds) {
#pragma unroll
      for (int i = 0; i < 16; ++i) Ssh[rr * SP + wave * 32 + acc_row(lane, i)] = from_f32<T>(st[i]);
    }
    __syncthreads();
    // (b) U = Uv - W S for this slice (two independent MFMA chains)
    if (makes_u) {
      f32x16 acc0 = {}, acc1 = {};
#pragma unroll
      for (int ks = 0; ks < DK / 16; ks += 2) {
        mfma_k16(acc0, wnow[ks], *(const F*)(Ssh + rr * SP + ks * 16 + h * 8));
        mfma_k16(acc1, wnow[ks + 1], *(const F*)(Ssh + rr * SP + (ks + 1) * 16 + h * 8));
      }
#pragma unroll
      for (int i = 0; i < 16; ++i)
        Ush[rr * UP + wave * 32 + acc_row(lane, i)] =
            from_f32<T>(to_f32(unow[i]) - (acc0[i] + acc1[i]));
    }
    __syncthreads();
    // (c) S = gamma_C S + Kt U
    if (holds) {
      f32x16 p0 = {}, p1 = {};
#pragma unroll
      for (int ks = 0; ks < C / 16; ks += 2) {
        mfma_k16(p0, know[ks], *(const F*)(Ush + rr * UP + ks * 16 + h * 8));
        mfma_k16(p1, know[ks + 1], *(const F*)(Ush + rr * UP + (ks + 1) * 16 + h * 8));
      }
#pragma unroll
      for (int i = 0; i < 16; ++i) st[i] = st[i] * gc + (p0[i] + p1[i]);
    }
  }
  if (holds) {
#pragma unroll
    for (int i = 0; i < 16; ++i) Sg[(int64_t)(wave * 32 + acc_row(lane, i)) * DV + sl + rr] = st[i];
  }
}

// Two-level scan kernels for dk = dv = 128: one block owns all 128 columns of its state (the
// Phi block or the Psi block of a segment, or the state in the combine), so every chunk's W and
// Kt are read once per block. Wave w keeps state rows [32 w, 32 w + 32) of all four column
// tiles; the U tiles (2 token tiles x 4 column tiles) are shared out two per wave.
template <typename T>
struct FullLds {
  static constexpr int C = gdr::C, P = gdr::PAD;
  static constexpr size_t ssh = 0;                                        // T[128][128+P]
  static constexpr size_t ush = ssh + (size_t)128 * (128 + P) * sizeof(T);  // T[128][C+P]
  static constexpr size_t bytes = ush + (size_t)128 * (C + P) * sizeof(T);
};

template <typename T>
__global__ __launch_bounds__(gdr::NT) void k_gdr_scan_seg(int Hv, int N, GdrWs ws) {
  using namespace gdr;
  typedef typename Frag8<T>::type F;
  typedef FullLds<T> L;
  constexpr int DK = 128, DV = 128, NCT = 4;  // column tiles of 32
  extern __shared__ __align__(16) unsigned char smem[];
  T* Ssh = (T*)(smem + L::ssh);  // [column][dk]
  T* Ush = (T*)(smem + L::ush);  // [column][token]
  constexpr int SP = DK + PAD, UP = C + PAD;
  const int P = ws.P;
  const bool phi = blockIdx.x == 0;
  const int hv = blockIdx.y, b = blockIdx.z / P, seg = blockIdx.z - b * P;
  const int NC = (N + C - 1) / C;
  const int c_begin = seg * ws.cps, c_end = min(NC, c_begin + ws.cps);
  const int64_t seq = (int64_t)b * Hv + hv;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int h = lane >> 5, rr = lane & 31;
  const int ut = wave & 1;        // token tile of this wave's U tiles
  const int uc0 = wave >> 1;      // its U column tiles: uc0 and uc0 + 2

  f32x16 st[NCT];
#pragma unroll
  for (int j = 0; j < NCT; ++j)
#pragma unroll
    for (int i = 0; i < 16; ++i)
      st[j][i] = (phi && wave * 32 + acc_row(lane, i) == j * 32 + rr) ? 1.f : 0.f;

  F wf[DK / 16], kf[C / 16];
  T uv[2][16];
  float gcn = 1.f;
  auto fetch = [&](int c) {
    const int64_t cid = seq * NC + c;
    gcn = ws.gc[cid];
    const T* W = ws.w<T>(cid, DK) + (int64_t)(ut * 32 + rr) * DK;
#pragma unroll
    for (int ks = 0; ks < DK / 16; ++ks) wf[ks] = *(const F*)(W + ks * 16 + h * 8);
    const T* Kt = ws.kt<T>(cid, DK) + (int64_t)(wave * 32 + rr) * C;
#pragma unroll
    for (int ks = 0; ks < C / 16; ++ks) kf[ks] = *(const F*)(Kt + ks * 16 + h * 8);
    if (!phi) {
      const T* Uv = ws.uv<T>(cid, DV) + (int64_t)(ut * 32) * DV + uc0 * 32 + rr;
#pragma unroll
      for (int q = 0; q < 2; ++q)
#pragma unroll
        for (int i = 0; i < 16; ++i) uv[q][i] = Uv[(int64_t)acc_row(lane, i) * DV + q * 64];
    }
  };
#pragma unroll
  for (int q = 0; q < 2; ++q)
#pragma unroll
    for (int i = 0; i < 16; ++i) uv[q][i] = from_f32<T>(0.f);
  if (c_begin < c_end) fetch(c_begin);
  for (int c = c_begin; c < c_end; ++c) {
    F wnow[DK / 16], know[C / 16];
    T unow[2][16];
#pragma unroll
    for (int q = 0; q < DK / 16; ++q) wnow[q] = wf[q];
#pragma unroll
    for (int q = 0; q < C / 16; ++q) know[q] = kf[q];
#pragma unroll
    for (int q = 0; q < 2; ++q)
#pragma unroll
      for (int i = 0; i < 16; ++i) unow[q][i] = uv[q][i];
    const float gc = gcn;
    if (c + 1 < c_end) fetch(c + 1);
    // (a) publish the state in the call dtype
#pragma unroll
    for (int j = 0; j < NCT; ++j)
#pragma unroll
      for (int i = 0; i < 16; ++i)
        Ssh[(j * 32 + rr) * SP + wave * 32 + acc_row(lane, i)] = from_f32<T>(st[j][i]);
    __syncthreads();
    // (b) U = Uv - W S: this wave's two tiles (token tile ut, column tiles uc0, uc0 + 2)
#pragma unroll
    for (int q = 0; q < 2; ++q) {
      const int uc = uc0 + 2 * q;
      f32x16 a0 = {}, a1 = {};
#pragma unroll
      for (int ks = 0; ks < DK / 16; ks += 2) {
        mfma_k16(a0, wnow[ks], *(const F*)(Ssh + (uc * 32 + rr) * SP + ks * 16 + h * 8));
        mfma_k16(a1, wnow[ks + 1], *(const F*)(Ssh + (uc * 32 + rr) * SP + (ks + 1) * 16 + h * 8));
      }
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        Ush[(uc * 32 + rr) * UP + ut * 32 + acc_row(lane, i)] =
            from_f32<T>(to_f32(unow[q][i]) - (a0[i] + a1[i]));
      }
    }
    __syncthreads();
    // (c) S = gamma_C S + Kt U for all four column tiles of this wave's rows
#pragma unroll
    for (int j = 0; j < NCT; ++j) {
      f32x16 p0 = {}, p1 = {};
#pragma unroll
      for (int ks = 0; ks < C / 16; ks += 2) {
        mfma_k16(p0, know[ks], *(const F*)(Ush + (j * 32 + rr) * UP + ks * 16 + h * 8));
        mfma_k16(p1, know[ks + 1], *(const F*)(Ush + (j * 32 + rr) * UP + (ks + 1) * 16 + h * 8));
      }
#pragma unroll
      for (int i = 0; i < 16; ++i) st[j][i] = st[j][i] * gc + (p0[i] + p1[i]);
    }
  }
  float* out = phi ? ws.phi + (seq * P + seg) * DK * DK : ws.psi + (seq * P + seg) * DK * DV;
#pragma unroll
  for (int j = 0; j < NCT; ++j)
#pragma unroll
    for (int i = 0; i < 16; ++i) out[(int64_t)(wave * 32 + acc_row(lane, i)) * 128 + j * 32 + rr] = st[j][i];
}

// S <- Phi_g S + Psi_g for g = 0 .. P-1, one block per (sequence, value head), all 128 columns.
template <typename T>
__global__ __launch_bounds__(gdr::NT) void k_gdr_combine_seg(float* __restrict__ S, int Hv, GdrWs ws) {
  using namespace gdr;
  typedef typename Frag8<T>::type F;
  typedef FullLds<T> L;
  constexpr int DK = 128, DV = 128, NCT = 4;
  extern __shared__ __align__(16) unsigned char smem[];
  T* Ssh = (T*)(smem + L::ssh);
  constexpr int SP = DK + PAD;
  const int P = ws.P;
  const int hv = blockIdx.y, b = blockIdx.z;
  const int64_t seq = (int64_t)b * Hv + hv;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int h = lane >> 5, rr = lane & 31;
  float* Sg = S + seq * DK * DV;
  f32x16 st[NCT];
#pragma unroll
  for (int j = 0; j < NCT; ++j)
#pragma unroll
    for (int i = 0; i < 16; ++i) st[j][i] = Sg[(int64_t)(wave * 32 + acc_row(lane, i)) * DV + j * 32 + rr];
  F af[DK / 16];
  auto fetch = [&](int g) {
    const float* Phi = ws.phi + (seq * P + g) * DK * DK + (int64_t)(wave * 32 + rr) * DK;
#pragma unroll
    for (int ks = 0; ks < DK / 16; ++ks) {
      const f32x4 lo = *(const f32x4*)(Phi + ks * 16 + h * 8);
      const f32x4 hi = *(const f32x4*)(Phi + ks * 16 + h * 8 + 4);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        af[ks][e] = from_f32<T>(lo[e]);
        af[ks][e + 4] = from_f32<T>(hi[e]);
      }
    }
  };
  fetch(0);
  for (int g = 0; g < P; ++g) {
    F anow[DK / 16];
#pragma unroll
    for (int q = 0; q < DK / 16; ++q) anow[q] = af[q];
    if (g + 1 < P) fetch(g + 1);
#pragma unroll
    for (int j = 0; j < NCT; ++j)
#pragma unroll
      for (int i = 0; i < 16; ++i)
        Ssh[(j * 32 + rr) * SP + wave * 32 + acc_row(lane, i)] = from_f32<T>(st[j][i]);
    __syncthreads();
    const float* Psi = ws.psi + (seq * P + g) * DK * DV;
#pragma unroll
    for (int j = 0; j < NCT; ++j) {
      f32x16 p0 = {}, p1 = {};
#pragma unroll
      for (int ks = 0; ks < DK / 16; ks += 2) {
        mfma_k16(p0, anow[ks], *(const F*)(Ssh + (j * 32 + rr) * SP + ks * 16 + h * 8));
        mfma_k16(p1, anow[ks + 1], *(const F*)(Ssh + (j * 32 + rr) * SP + (ks + 1) * 16 + h * 8));
      }
#pragma unroll
      for (int i = 0; i < 16; ++i)
        st[j][i] = (p0[i] + p1[i]) + Psi[(int64_t)(wave * 32 + acc_row(lane, i)) * DV + j * 32 + rr];
    }
    __syncthreads();  // every wave is done reading Ssh before the next step rewrites it
  }
#pragma unroll
  for (int j = 0; j < NCT; ++j)
#pragma unroll
    for (int i = 0; i < 16; ++i) Sg[(int64_t)(wave * 32 + acc_row(lane, i)) * DV + j * 32 + rr] = st[j][i];
}

template <typename K>
static void allow_lds_bytes(K kernel, size_t bytes) {
  (void)hipFuncSetAttribute((const void*)kernel, hipFuncAttributeMaxDynamicSharedMemorySize,
                            (int)bytes);
}

template <typename T, int DK, int DV>
static hipError_t gdr_launch(const void* k, const void* v, const float* alpha, const float* beta,
                             float* S, int B, int Hk, int Hv, int N, GdrWs ws, hipStream_t s,
                             const LaunchEvents& ev) {
  typedef GdrLds<T, DK, DV> LP;
  typedef ScanLds<T, DK> LS;
  static bool once = [] {
    allow_lds_bytes(k_gdr_prep<T, DK, DV>, LP::bytes);
    allow_lds_bytes(k_gdr_scan<T, DK, DV>, LS::bytes);
    if constexpr (DK == 128 && DV == 128) {
      allow_lds_bytes(k_gdr_scan_seg<T>, FullLds<T>::bytes);
      allow_lds_bytes(k_gdr_combine_seg<T>, FullLds<T>::bytes);
    }
    return true;
  }();
  (void)once;
  const int NC = (N + gdr::C - 1) / gdr::C;
  record(ev.gdr_prep[0], s);
  k_gdr_prep<T, DK, DV><<<dim3(NC, Hv, B), gdr::NT, LP::bytes, s>>>(
      (const T*)k, (const T*)v, alpha, beta, Hk, Hv, N, ws);
  record(ev.gdr_prep[1], s);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  record(ev.gdr_scan[0], s);
  if (ws.P > 1) {
    if constexpr (DK == 128 && DV == 128) {
      k_gdr_scan_seg<T><<<dim3(2, Hv, B * ws.P), gdr::NT, FullLds<T>::bytes, s>>>(Hv, N, ws);
      e = hipGetLastError();
      if (e != hipSuccess) return e;
      k_gdr_combine_seg<T><<<dim3(1, Hv, B), gdr::NT, FullLds<T>::bytes, s>>>(S, Hv, ws);
    } else {
      return hipErrorInvalidValue;  // segments are only planned for dk = dv = 128
    }
  } else {
    k_gdr_scan<T, DK, DV><<<dim3(DV / 32, Hv, B), gdr::NT, LS::bytes, s>>>(S, Hv, N, ws);
  }
  record(ev.gdr_scan[1], s);
  return hipGetLastError();
}

// Segments of the two-level scan, from a latency model of the two schedules (times per chunk
// step measured on MI355X at dk = dv = 128): the plain scan runs every chunk in order at about
// 1.5 us a step with DV / 32 small blocks per sequence; the segmented scan runs ceil(NC / P)
// steps at about 3.4 us, in as many rounds as its 2 B Hv P one-per-CU blocks need, and the
// combine adds P steps of about 3.7 us. P = 1 selects the plain scan. The scan's grid dimension
// B * P stays within 65535.
static void gdr_segments(int NC, int B, int Hv, int dk, int dv, int& P, int& cps) {
  P = 1;
  cps = NC;
  if (dk != 128 || dv != 128 || NC < 16) return;
  const double cus = 256.0;
  const double plain_rounds = std::ceil(B * (double)Hv * (dv / 32) / (cus * 8));
  double best = plain_rounds * NC * 1.5;
  const int pmax = std::min(64, std::min(NC / 2, 65535 / B));
  for (int p = 2; p <= pmax; ++p) {
    const int c = (NC + p - 1) / p;
    const int pp = (NC + c - 1) / c;
    const double rounds = std::ceil(2.0 * B * Hv * pp / cus);
    const double t = rounds * c * 3.4 + pp * 3.7 * std::ceil(B * (double)Hv / cus);
    if (t < best) {
      best = t;
      P = pp;
      cps = c;
    }
  }
}

GdrWs gdr_layout(void* base, int B, int Hv, int N, int dk, int dv, int dtype) {
  const size_t e = dtype == 1 ? 2 : 4;
  const int NC = (N + gdr::C - 1) / gdr::C;
  const int64_t chunks = (int64_t)B * Hv * NC;
  auto al = [](size_t x) { return (x + 255) / 256 * 256; };
  GdrWs w{};
  gdr_segments(NC, B, Hv, dk, dv, w.P, w.cps);
  char* p = (char*)base;
  size_t o = 0;
  w.w_ = p ? p + o : nullptr;   o += al((size_t)chunks * gdr::C * dk * e);
  w.uv_ = p ? p + o : nullptr;  o += al((size_t)chunks * gdr::C * dv * e);
  w.kt_ = p ? p + o : nullptr;  o += al((size_t)chunks * gdr::C * dk * e);
  w.gc = p ? (float*)(p + o) : nullptr;
  o += al((size_t)chunks * 4);
  const size_t segs = w.P > 1 ? (size_t)B * Hv * w.P : 0;
  w.phi = p ? (float*)(p + o) : nullptr;  o += al(segs * dk * dk * 4);
  w.psi = p ? (float*)(p + o) : nullptr;  o += al(segs * dk * dv * 4);
  w.bytes = o;
  return w;
}

hipError_t launch_delta_rule(const void* k, const void* v, const float* alpha, const float* beta,
                             float* S, int B, int Hk, int Hv, int N, int dk, int dv, int dtype,
                             GdrWs ws, hipStream_t s, const LaunchEvents& ev) {
  if (dtype == 1) {
    if (dk == 128 && dv == 128) return gdr_launch<bf16, 128, 128>(k, v, alpha, beta, S, B, Hk, Hv, N, ws, s, ev);
    if (dk == 128 && dv == 64) return gdr_launch<bf16, 128, 64>(k, v, alpha, beta, S, B, Hk, Hv, N, ws, s, ev);
    if (dk == 64 && dv == 128) return gdr_launch<bf16, 64, 128>(k, v, alpha, beta, S, B, Hk, Hv, N, ws, s, ev);
    return gdr_launch<bf16, 64, 64>(k, v, alpha, beta, S, B, Hk, Hv, N, ws, s, ev);
  }
  if (dk == 128 && dv == 128) return gdr_launch<float, 128, 128>(k, v, alpha, beta, S, B, Hk, Hv, N, ws, s, ev);
  if (dk == 128 && dv == 64) return gdr_launch<float, 128, 64>(k, v, alpha, beta, S, B, Hk, Hv, N, ws, s, ev);
  if (dk == 64 && dv == 128) return gdr_launch<float, 64, 128>(k, v, alpha, beta, S, B, Hk, Hv, N, ws, s, ev);
  return gdr_launch<float, 64, 64>(k, v, alpha, beta, S, B, Hk, Hv, N, ws, s, ev);
}

}  // namespace dv
