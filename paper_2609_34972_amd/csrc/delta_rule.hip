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

#include <cfloat>

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
  k_gdr_scan<T, DK, DV><<<dim3(DV / 32, Hv, B), gdr::NT, LS::bytes, s>>>(S, Hv, N, ws);
  record(ev.gdr_scan[1], s);
  return hipGetLastError();
}

GdrWs gdr_layout(void* base, int B, int Hv, int N, int dk, int dv, int dtype) {
  const size_t e = dtype == 1 ? 2 : 4;
  const int64_t chunks = (int64_t)B * Hv * ((N + gdr::C - 1) / gdr::C);
  auto al = [](size_t x) { return (x + 255) / 256 * 256; };
  GdrWs w{};
  char* p = (char*)base;
  size_t o = 0;
  w.w_ = p ? p + o : nullptr;   o += al((size_t)chunks * gdr::C * dk * e);
  w.uv_ = p ? p + o : nullptr;  o += al((size_t)chunks * gdr::C * dv * e);
  w.kt_ = p ? p + o : nullptr;  o += al((size_t)chunks * gdr::C * dk * e);
  w.gc = p ? (float*)(p + o) : nullptr;
  o += al((size_t)chunks * 4);
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
