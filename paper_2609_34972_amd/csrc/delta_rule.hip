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
// the two products, fp32 forward substitution for T) and stores them as one record per chunk
// in fragment order (below). k_gdr_chain then runs the chunks in order, U = Uv - W S and
// S = gamma_C S + Kt U. The rule acts on every state column independently: each wave keeps 32
// columns of the fp32 state, all dk rows, in MFMA accumulators, and since those accumulators
// (and those of U) are already the B operands of the next product in a permuted k order, a
// wave's chain needs no exchange with other waves; the block only shares the chunk record,
// copied into LDS one chunk ahead. Products read the state rounded to the call dtype; the
// state itself stays fp32.
//
// Long sequences use a two-level scan. The chunk step is affine in S, so a run of chunks maps
// a start state S to Phi S + Psi: the segments of ws.cps chunks run at once, from the start
// state I for Phi (without Uv) and 0 for Psi (segment 0 from S itself), and k_gdr_merge then
// applies them in order.
#include "delta_rule.hpp"

#include <algorithm>
#include <cfloat>
#include <cmath>

#include "dv_device.hpp"
#include "gemm_pipe.hpp"

namespace dv {

namespace gdr {
constexpr int C = 64;     // tokens per chunk
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

// Fragment order. One 32x32x16 MFMA step takes from lane half h the 8 values at k = 8 h .. 8 h + 7
// of its row (A) or column (B); any assignment of the 16 k to (half, slot) pairs works as long as
// both operands use it. A 32x32 accumulator tile holds in lane half h, items 8 q .. 8 q + 7, the
// rows 16 q + {4 h .. 4 h + 3, 8 + 4 h .. 8 + 4 h + 3}: so with k assigned the same way, items
// 8 q .. 8 q + 7 of an accumulator are directly the B fragment of k step q. Matrices meant to
// meet such accumulators store every row with the index m inside each 16-group moved to
// position frag_pos(m) (bits 2 and 3 swapped, an involution), so that a lane half's 8 values
// are contiguous; the 16-byte chunks of a row are XOR-swizzled by the row so that the 16 rows
// one fragment load touches fall in distinct LDS bank groups.
__device__ __forceinline__ int frag_pos(int m) { return (m & ~12) | ((m & 4) << 1) | ((m & 8) >> 1); }

// Element offset of logical position pos in row `row` of a fragment-order matrix of INNER
// values per row.
template <typename T, int INNER>
__device__ __forceinline__ int frag_off(int row, int pos) {
  constexpr int EPC = 16 / (int)sizeof(T), CPR = INNER / EPC;
  static_assert(CPR == 8 || CPR == 16 || CPR == 32, "row of 8, 16 or 32 chunks");
  const int key = CPR >= 16 ? (row & 15) : ((row >> 1) & 7);
  return row * INNER + (((pos / EPC) ^ key) * EPC) + pos % EPC;
}

// The 8 values at logical positions 8 g .. 8 g + 7 of row `row`.
template <typename T, int INNER>
__device__ __forceinline__ typename Frag8<T>::type frag_get(const T* m, int row, int g) {
  typedef typename Frag8<T>::type F;
  if constexpr (sizeof(T) == 2) {
    return *(const F*)(m + frag_off<T, INNER>(row, 8 * g));
  } else {
    const f32x4 lo = *(const f32x4*)(m + frag_off<T, INNER>(row, 8 * g));
    const f32x4 hi = *(const f32x4*)(m + frag_off<T, INNER>(row, 8 * g + 4));
    return F{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
  }
}

template <typename T, int INNER>
__device__ __forceinline__ void frag_put(T* m, int row, int g, typename Frag8<T>::type x) {
  typedef typename Frag8<T>::type F;
  if constexpr (sizeof(T) == 2) {
    *(F*)(m + frag_off<T, INNER>(row, 8 * g)) = x;
  } else {
    *(f32x4*)(m + frag_off<T, INNER>(row, 8 * g)) = f32x4{x[0], x[1], x[2], x[3]};
    *(f32x4*)(m + frag_off<T, INNER>(row, 8 * g + 4)) = f32x4{x[4], x[5], x[6], x[7]};
  }
}

// Items 8 q .. 8 q + 7 of an accumulator tile, rounded to T: a B fragment in fragment order.
template <typename T>
__device__ __forceinline__ typename Frag8<T>::type acc_frag(const f32x16& a, int q) {
  typename Frag8<T>::type x;
#pragma unroll
  for (int e = 0; e < 8; ++e) x[e] = from_f32<T>(a[8 * q + e]);
  return x;
}

// Per-chunk record of the workspace: -W [C][DK], Kt [DK][C], Uv^T [DV][C], all in fragment order.
template <typename T, int DK, int DV>
struct GdrRec {
  static constexpr int C = gdr::C;
  static constexpr int KT = C * DK, UV = 2 * C * DK, ELEMS = C * (2 * DK + DV);
};

// The chunk's K and V transposed in LDS ([channel][token], 64 tokens a row): 16-byte chunks of a
// row XOR-swizzled by the row, so that the 16 rows one fragment load touches fall in distinct
// bank groups without padding.
template <typename T>
__device__ __forceinline__ int vk_off(int n, int s) {
  constexpr int EPC = 16 / (int)sizeof(T), CPR = gdr::C / EPC;
  const int key = CPR >= 16 ? (n & 15) : ((n >> 1) & 7);
  return n * gdr::C + (((s / EPC) ^ key) * EPC) + s % EPC;
}

// 8 consecutive tokens s0 .. s0 + 7 (s0 a multiple of 8) of row n.
template <typename T>
__device__ __forceinline__ typename Frag8<T>::type vk_frag(const T* m, int n, int s0) {
  typedef typename Frag8<T>::type F;
  if constexpr (sizeof(T) == 2) {
    return *(const F*)(m + vk_off<T>(n, s0));
  } else {
    const f32x4 lo = *(const f32x4*)(m + vk_off<T>(n, s0));
    const f32x4 hi = *(const f32x4*)(m + vk_off<T>(n, s0 + 4));
    return F{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
  }
}

// LDS layout of k_gdr_prep (byte offsets). M holds A and is turned into T = (I + A)^-1 in place;
// the bf16 block stays under 53 KiB so that three share a CU.
template <typename T, int DK, int DV>
struct GdrLds {
  static constexpr int C = gdr::C;
  static constexpr int MP = C + 4;                                 // fp32 pitch of M (bank spread)
  static constexpr size_t g = 0;                                   // float[C]  g_t
  static constexpr size_t beta = g + C * 4;                        // float[C]  beta_t
  static constexpr size_t bg = beta + C * 4;                       // float[C]  beta_t gamma_t
  static constexpr size_t m = bg + C * 4;                          // float[C][MP]
  static constexpr size_t vt = m + (size_t)C * MP * 4;             // T[DV][C]  V^T
  static constexpr size_t kt = vt + (size_t)DV * C * sizeof(T);    // T[DK][C]  K^T
  static constexpr size_t bytes = kt + (size_t)DK * C * sizeof(T);
};

// D[16x16] += A[16x4] B[4x16] in fp32; lane l gives A[l % 16][l / 16] and B[l / 16][l % 16] and
// holds D[4 (l / 16) + r][l % 16] in item r.
__device__ __forceinline__ void mfma16x4(f32x4& d, float a, float b) {
  d = __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, d, 0, 0, 0);
}

// out[16x16] = X[16 x 4 nk] Y[4 nk x 16] for fp32 matrices in M (pitch MP); X rows from xr, its
// columns from xc; Y rows from yr, its columns from yc; k runs over 4 k0 .. 4 (k0 + nk) - 1.
template <int MP>
__device__ __forceinline__ f32x4 mm16(const float* M, int xr, int xc, int yr, int yc, int k0, int nk) {
  const int lane = threadIdx.x & 63, i = lane & 15, kk = lane >> 4;
  f32x4 d = {};
  for (int ks = k0; ks < k0 + nk; ++ks)
    mfma16x4(d, M[(xr + i) * MP + xc + 4 * ks + kk], M[(yr + 4 * ks + kk) * MP + yc + i]);
  return d;
}

template <int MP>
__device__ __forceinline__ void put16(float* M, int r0, int c0, f32x4 d, float sign) {
  const int lane = threadIdx.x & 63;
#pragma unroll
  for (int r = 0; r < 4; ++r) M[(r0 + 4 * (lane >> 4) + r) * MP + c0 + (lane & 15)] = sign * d[r];
}

template <typename T, int DK, int DV>
__global__ __launch_bounds__(gdr::NT) void k_gdr_prep(const T* __restrict__ k,
                                                      const T* __restrict__ v,
                                                      const float* __restrict__ alpha,
                                                      const float* __restrict__ beta, int Hk,
                                                      int Hv, int N, GdrWs ws) {
  using namespace gdr;
  typedef GdrLds<T, DK, DV> L;
  typedef typename Frag8<T>::type F;
  constexpr int MP = L::MP;
  extern __shared__ __align__(16) unsigned char smem[];
  float* g = (float*)(smem + L::g);
  float* bet = (float*)(smem + L::beta);
  float* bgm = (float*)(smem + L::bg);
  float* M = (float*)(smem + L::m);
  T* VT = (T*)(smem + L::vt);
  T* KT = (T*)(smem + L::kt);

  const int c = blockIdx.x, hv = blockIdx.y, b = blockIdx.z;
  const int NC = (N + C - 1) / C;
  const int hk = hv / (Hv / Hk);
  const int64_t t0 = (int64_t)c * C;
  const int nval = (int)min((int64_t)C, (int64_t)N - t0);
  const int64_t seq = (int64_t)b * Hv + hv;  // (sequence, value head)
  const T* kc = k + (((int64_t)b * Hk + hk) * N + t0) * DK;
  const T* vc = v + (seq * N + t0) * DV;
  const int tid = threadIdx.x, lane = tid & 63, wave = wave_index();
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
    bgm[lane] = be * __expf(x);
  }
  // 2. The chunk's K and V, transposed into LDS (B operands of the two products, and the rows
  //    of Kt).
#pragma unroll
  for (int q = 0; q < VP; ++q) {
    const int idx = tid + q * NT, sidx = idx % C, n0 = (idx / C) * 8;
#pragma unroll
    for (int e = 0; e < 8; ++e) VT[vk_off<T>(n0 + e, sidx)] = vpc[q][e];
  }
#pragma unroll
  for (int q = 0; q < KP; ++q) {
    const int idx = tid + q * NT, sidx = idx % C, n0 = (idx / C) * 8;
#pragma unroll
    for (int e = 0; e < 8; ++e) KT[vk_off<T>(n0 + e, sidx)] = kpc[q][e];
  }
  __syncthreads();
  const float gC = g[C - 1];

  // 3. A[t][s] = beta_t exp(g_t - g_s) k_t.k_s for s < t (K K^T on MFMA, lower tiles only; the
  //    upper right tile of M is never read as part of A or T).
  if (wave < 3) {
    f32x16 acc = {};
#pragma unroll
    for (int ks = 0; ks < DK / 16; ++ks) mfma_k16(acc, fa3[ks], fb3[ks]);
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int t = ti3 * 32 + acc_row(lane, i), sx = si3 * 32 + rr;
      M[t * MP + sx] = sx < t ? bet[t] * __expf(g[t] - g[sx]) * acc[i] : 0.f;
    }
  }
  __syncthreads();

  // 4. T = (I + A)^-1 for the unit lower-triangular I + A, in place, by 2 x 2 block recursion
  //    over 16 x 16 blocks D_0..D_3 on the diagonal:
  //      level 0: D_b = (I + A_bb)^-1 by forward substitution (wave 0: lane 16 b + j runs
  //               column j of D_b, the column in registers, rows of A read as LDS broadcasts
  //               and summed in four chains; each row is read before it is overwritten);
  //      level 1: in each 32 x 32 block p, T_(2p+1)(2p) = -D_(2p+1) (A_(2p+1)(2p) D_(2p));
  //      level 2: T21 = -T22 (A21 T11).
  //    Products run on fp32 MFMA (16x16x4), their intermediates in the upper right 32 x 32 block
  //    of M, which the chunk's products never read. Meanwhile waves 1..3 write Kt.
  if (wave == 0) {
    const int o = (lane >> 4) * 16, j = lane & 15;
    float col[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      float x4[4] = {0.f, 0.f, 0.f, 0.f};
      const float* arow = M + (o + i) * MP + o;
#pragma unroll
      for (int s4 = 0; s4 < i; s4 += 4) {
        const f32x4 a4 = *(const f32x4*)(arow + s4);
#pragma unroll
        for (int u = 0; u < 4; ++u)
          if (s4 + u < i) x4[u] -= a4[u] * col[s4 + u];
      }
      const float x = (x4[0] + x4[1]) + (x4[2] + x4[3]);
      col[i] = i < j ? 0.f : (i == j ? 1.f : x);
      M[(o + i) * MP + o + j] = col[i];
    }
  } else {
    // Kt in fragment order: logical positions 8 gq .. 8 gq + 7 of row n hold tokens
    // frag_pos(8 gq + e), two runs of four.
    T* Kt = ws.rec<T>(seq * NC + c) + GdrRec<T, DK, DV>::KT;
    for (int idx = tid - 64; idx < DK * (C / 8); idx += NT - 64) {
      const int n = idx / (C / 8), gq = idx % (C / 8);
      const int tq = (gq >> 1) * 16 + (gq & 1) * 4;
      F y;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const int t = tq + (e >> 2) * 8 + (e & 3);
        y[e] = from_f32<T>(__expf(gC - g[t]) * to_f32(KT[vk_off<T>(n, t)]));
      }
      frag_put<T, C>(Kt, n, gq, y);
    }
  }
  __syncthreads();
  if (wave < 2) {  // level 1, block p = wave; scratch Y_p at rows 16 p.., columns 32..47
    const int p = wave, o = 32 * p;
    put16<MP>(M, 16 * p, 32, mm16<MP>(M, o + 16, o, o, o, 0, 4), 1.f);
    put16<MP>(M, o + 16, o, mm16<MP>(M, o + 16, o + 16, 16 * p, 32, 0, 4), -1.f);
  }
  __syncthreads();
  {  // level 2, X = A21 T11: tile (a, bb) of the 32 x 32 result per wave, to rows 0..31,
     // columns 32..63 (T11 is lower triangular: k from 16 bb)
    const int a = wave >> 1, bb = wave & 1;
    put16<MP>(M, 16 * a, 32 + 16 * bb, mm16<MP>(M, 32 + 16 * a, 0, 0, 16 * bb, 4 * bb, 8 - 4 * bb), 1.f);
  }
  __syncthreads();
  {  // T21 = -T22 X over A21's place (T22 is lower triangular: k up to 16 a + 15)
    const int a = wave >> 1, bb = wave & 1;
    put16<MP>(M, 32 + 16 * a, 16 * bb, mm16<MP>(M, 32 + 16 * a, 32, 0, 32 + 16 * bb, 0, 4 + 4 * a), -1.f);
  }
  __syncthreads();

  // 5. Uv = (T diag(beta)) V and W = (T diag(beta gamma)) K: waves 0, 1 the Uv row tiles 0, 1 and
  //    waves 2, 3 the W row tiles, each over every column tile. The scaled rows of T are formed
  //    in the call dtype as they are read (row tile 0 of T is zero beyond column 31). Uv comes
  //    out with a value column per lane and W, computed as K^T (T diag(beta gamma))^T, with a
  //    token per lane, so both store rows of their fragment-order form (Uv^T and -W): items
  //    8 q .. 8 q + 7 of a tile are logical positions 16 q + 8 h .. + 7 of the lane's row.
  {
    const bool isu = wave < 2;
    const int ti = wave & 1, nks = ti == 0 ? 2 : 4;
    const float* sc = isu ? bet : bgm;
    F tf[4];
#pragma unroll
    for (int ks = 0; ks < 4; ++ks) {
      if (ks < nks) {
        const float* row = M + (ti * 32 + rr) * MP + ks * 16 + h * 8;
        const f32x4 lo = *(const f32x4*)row, hi = *(const f32x4*)(row + 4);
        const f32x4 slo = *(const f32x4*)(sc + ks * 16 + h * 8), shi = *(const f32x4*)(sc + ks * 16 + h * 8 + 4);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          tf[ks][e] = from_f32<T>(lo[e] * slo[e]);
          tf[ks][e + 4] = from_f32<T>(hi[e] * shi[e]);
        }
      }
    }
    T* rec = ws.rec<T>(seq * NC + c);
    const int nd = isu ? DV / 32 : DK / 32;
    for (int ni = 0; ni < nd; ++ni) {
      f32x16 acc = {};
#pragma unroll
      for (int ks = 0; ks < 4; ++ks) {
        if (ks < nks) {
          if (isu)
            mfma_k16(acc, tf[ks], vk_frag<T>(VT, ni * 32 + rr, ks * 16 + h * 8));
          else
            mfma_k16(acc, vk_frag<T>(KT, ni * 32 + rr, ks * 16 + h * 8), tf[ks]);
        }
      }
      if (isu) {
#pragma unroll
        for (int qh = 0; qh < 2; ++qh)
          frag_put<T, C>(rec + GdrRec<T, DK, DV>::UV, ni * 32 + rr, ti * 4 + 2 * qh + h, acc_frag<T>(acc, qh));
      } else {
#pragma unroll
        for (int qh = 0; qh < 2; ++qh)
          frag_put<T, DK>(rec, ti * 32 + rr, ni * 4 + 2 * qh + h, acc_frag<T>(-acc, qh));
      }
    }
  }
  if (tid == 0) ws.gc[seq * NC + c] = __expf(gC);
}

// Offset of Phi[i][j] in a segment's transition matrix: fp32 rows of DK, 16-byte chunks XOR-
// swizzled by the row, so that k_gdr_merge can copy the matrix into LDS as it is and read A
// fragments (a row, two runs of four columns) without bank conflicts.
template <int DK>
__device__ __forceinline__ int phi_off(int i, int j) {
  return i * DK + (((j >> 2) ^ (i & 15)) << 2) + (j & 3);
}

// LDS of k_gdr_chain: the chunk records in NS buffers (bf16: three, so that two records are in
// flight while one is used; fp32: one). Per wave, a record copy is INS_PSI (with Uv) or INS_PHI
// (without) 1 KiB instructions.
template <typename T, int DK, int DV>
struct ChainLds {
  typedef GdrRec<T, DK, DV> R;
  static constexpr int NS = sizeof(T) == 2 ? 3 : 1;
  static constexpr size_t bytes = (size_t)NS * R::ELEMS * sizeof(T);
  static constexpr int INS_PSI = R::ELEMS * (int)sizeof(T) / 1024 / (gdr::NT / 64);
  static constexpr int INS_PHI = R::UV * (int)sizeof(T) / 1024 / (gdr::NT / 64);
  static_assert(R::ELEMS * sizeof(T) % (1024 * (gdr::NT / 64)) == 0 && R::UV * sizeof(T) % (1024 * (gdr::NT / 64)) == 0,
                "every wave copies the same number of KiB");
  static_assert(bytes <= 160 * 1024 && INS_PSI < 64, "fits LDS and the vmcnt counter");
};

// Copies one chunk record (a multiple of 1 KiB) into LDS, 1 KiB per wave instruction, waves
// taking every fourth KiB. Straight into LDS: nothing passes through registers.
__device__ __forceinline__ void gdr_copy_record(const void* src, int bytes, unsigned char* dst, int wave, int nins) {
  const auto rs = buffer_rsrc(src, bytes);
  const int lane = threadIdx.x & 63;
  for (int blk = wave; blk < nins; blk += gdr::NT / 64)
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_void*)(dst + blk * 1024), 16, lane * 16, blk * 1024, 0, 0);
}

// Column blocks of 128 state columns.
constexpr int gdr_xblocks(int cols) { return (cols + 127) / 128; }

// The chunks of one segment (the whole sequence when ws.P == 1) in order for one (sequence,
// value head): grid (column blocks, Hv, B * P). With P > 1 the first gdr_xblocks(DK) column
// blocks carry the columns of Phi, the others those of Psi. Each wave owns 32 columns.
template <typename T, int DK, int DV>
__global__ __launch_bounds__(gdr::NT) __attribute__((amdgpu_waves_per_eu(1, 1))) void k_gdr_chain(float* __restrict__ S, const float* __restrict__ gcs, int Hv, int N, GdrWs ws) {
  using namespace gdr;
  typedef GdrRec<T, DK, DV> R;
  typedef ChainLds<T, DK, DV> L;
  constexpr int NKT = DK / 32, XPHI = gdr_xblocks(DK);
  extern __shared__ __align__(16) unsigned char smem[];
  const int P = ws.P;
  const int hv = blockIdx.y, b = blockIdx.z / P, seg = blockIdx.z - b * P;
  const bool phi = P > 1 && (int)blockIdx.x < XPHI;
  if (phi && seg == 0) return;  // segment 0 starts from S itself: no transition matrix needed
  const int xb = P > 1 && !phi ? blockIdx.x - XPHI : blockIdx.x;
  const int ncols = phi ? DK : DV;
  const int NC = (N + C - 1) / C;
  const int c_begin = seg * ws.cps, c_end = min(NC, c_begin + ws.cps);
  const int64_t seq = (int64_t)b * Hv + hv;
  const int lane = threadIdx.x & 63, wave = wave_index();
  const int h = lane >> 5, rr = lane & 31;
  const int n0 = xb * 128 + wave * 32;  // first column of this wave
  const bool active = n0 < ncols;
  const bool from_s = P == 1 || (!phi && seg == 0);
  const bool uses_uv = !phi;
  const int copy_bytes = (uses_uv ? R::ELEMS : R::UV) * (int)sizeof(T);
  const int nins = copy_bytes / 1024;  // 1 KiB per wave instruction (64 lanes x 16 bytes)

  f32x16 st[NKT];
#pragma unroll
  for (int kt = 0; kt < NKT; ++kt) st[kt] = f32x16{};
  if (active) {
    if (from_s) {
      const float* Sg = S + seq * DK * DV + n0 + rr;
#pragma unroll
      for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
        for (int i = 0; i < 16; ++i) st[kt][i] = Sg[(int64_t)(kt * 32 + acc_row(lane, i)) * DV];
    } else if (phi) {
#pragma unroll
      for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
        for (int i = 0; i < 16; ++i) st[kt][i] = kt * 32 + acc_row(lane, i) == n0 + rr ? 1.f : 0.f;
    }
  }

  auto issue = [&](int c, int stage) {
    gdr_copy_record(ws.rec<T>(seq * NC + c), copy_bytes, smem + (size_t)stage * R::ELEMS * sizeof(T), wave, nins);
  };

  issue(c_begin, 0);
  if (L::NS == 3 && c_begin + 1 < c_end) issue(c_begin + 1, 1);
  int stage = 0;
  for (int c = c_begin; c < c_end; ++c) {
    const float gc = gcs[seq * NC + c];
    // This wave's copies of chunk c have landed (those of chunk c + 1, issued after them, may
    // still be in flight); the barrier makes that true of every wave and ends every wave's reads
    // of the buffer that chunk c + 2 goes to.
    if (L::NS == 3 && c + 1 < c_end) {
      if (uses_uv)
        pipe_sync<waitcnt_imm(L::INS_PSI, 0)>();
      else
        pipe_sync<waitcnt_imm(L::INS_PHI, 0)>();
    } else {
      pipe_sync<waitcnt_imm(0, 0)>();
    }
    if (L::NS == 3 && c + 2 < c_end) issue(c + 2, stage == 0 ? 2 : stage - 1);
    if (active) {
      typedef typename Frag8<T>::type F;
      const T* Wn = (const T*)(smem + (size_t)stage * R::ELEMS * sizeof(T));
      const T* Kt = Wn + R::KT;
      const T* UvT = Wn + R::UV;
      // Every fragment of the step is read up front (one block per CU leaves the registers
      // for it), so that LDS latency is paid once per phase, not once per MFMA.
      F wf[2][NKT][2], uf[2][2];
#pragma unroll
      for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
        for (int q = 0; q < 2; ++q)
#pragma unroll
          for (int tt = 0; tt < 2; ++tt) wf[tt][kt][q] = frag_get<T, DK>(Wn, tt * 32 + rr, kt * 4 + 2 * q + h);
      // (read in Phi blocks too, where the buffer's Uv part is stale: the values are not used)
#pragma unroll
      for (int tt = 0; tt < 2; ++tt)
#pragma unroll
        for (int q = 0; q < 2; ++q) uf[tt][q] = frag_get<T, C>(UvT, n0 + rr, tt * 4 + 2 * q + h);
      // U = Uv - W S for the two token tiles (the record holds -W); S enters rounded to T
      F sb[NKT][2];
#pragma unroll
      for (int kt = 0; kt < NKT; ++kt) {
        sb[kt][0] = acc_frag<T>(st[kt], 0);
        sb[kt][1] = acc_frag<T>(st[kt], 1);
      }
      f32x16 u[2];
#pragma unroll
      for (int tt = 0; tt < 2; ++tt)
#pragma unroll
        for (int q = 0; q < 2; ++q)
#pragma unroll
          for (int e = 0; e < 8; ++e) u[tt][8 * q + e] = uses_uv ? to_f32(uf[tt][q][e]) : 0.f;
#pragma unroll
      for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
        for (int q = 0; q < 2; ++q)
#pragma unroll
          for (int tt = 0; tt < 2; ++tt) mfma_k16(u[tt], wf[tt][kt][q], sb[kt][q]);
      // S = gamma_C S + Kt U
      F kf[NKT][2][2];
#pragma unroll
      for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
        for (int tt = 0; tt < 2; ++tt)
#pragma unroll
          for (int q = 0; q < 2; ++q) kf[kt][tt][q] = frag_get<T, C>(Kt, kt * 32 + rr, tt * 4 + 2 * q + h);
#pragma unroll
      for (int kt = 0; kt < NKT; ++kt) st[kt] *= gc;
      F ub[2][2];
#pragma unroll
      for (int tt = 0; tt < 2; ++tt) {
        ub[tt][0] = acc_frag<T>(u[tt], 0);
        ub[tt][1] = acc_frag<T>(u[tt], 1);
      }
#pragma unroll
      for (int tt = 0; tt < 2; ++tt)
#pragma unroll
        for (int q = 0; q < 2; ++q)
#pragma unroll
          for (int kt = 0; kt < NKT; ++kt) mfma_k16(st[kt], kf[kt][tt][q], ub[tt][q]);
      // Schedule: the W and Uv reads first, then the U products with the Kt reads between them
      // (they land while the products run), then the state products.
      if constexpr (sizeof(T) == 2) {
        __builtin_amdgcn_sched_group_barrier(0x100, 4 * NKT + 4, 0);
#pragma unroll
        for (int i = 0; i < 4 * NKT; ++i) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
          __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        }
        __builtin_amdgcn_sched_group_barrier(0x008, 4 * NKT, 0);
      }
    }
    if (L::NS == 1 && c + 1 < c_end) {
      __syncthreads();
      issue(c + 1, 0);
    }
    stage = L::NS == 3 ? (stage == 2 ? 0 : stage + 1) : 0;
  }
  if (!active) return;
  if (phi) {
    float* out = ws.phi + (seq * P + seg) * DK * DK;
#pragma unroll
    for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
      for (int i = 0; i < 16; ++i) out[phi_off<DK>(kt * 32 + acc_row(lane, i), n0 + rr)] = st[kt][i];
    return;
  }
  float* out = P == 1 ? S + seq * DK * DV : ws.psi + (seq * P + seg) * DK * DV;
#pragma unroll
  for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
    for (int i = 0; i < 16; ++i) out[(int64_t)(kt * 32 + acc_row(lane, i)) * DV + n0 + rr] = st[kt][i];
}

// S <- Phi_g S + Psi_g for g = 1 .. P-1, from S = Psi_0; grid (column blocks, Hv, B), 32 state
// columns per wave. The block copies each Phi_g into LDS once (two buffers, the next one in
// flight) and every wave reads it as the A operand in the k order of the state's accumulators,
// rounded to the call dtype as the chunk steps round their operands. Psi_g is loaded one step
// ahead, before the next copy is issued, so that waiting for it never waits for the copy.
template <typename T, int DK>
struct MergeLds {
  static constexpr int PHI_BYTES = DK * DK * 4;
  static constexpr size_t bytes = 2 * (size_t)PHI_BYTES;
  static constexpr int INS = PHI_BYTES / 1024 / (gdr::NT / 64);
  static_assert(PHI_BYTES % (1024 * (gdr::NT / 64)) == 0, "every wave copies the same number of KiB");
};

template <typename T, int DK, int DV>
__global__ __launch_bounds__(gdr::NT) void k_gdr_merge(float* __restrict__ S, int Hv, GdrWs ws) {
  typedef typename Frag8<T>::type F;
  typedef MergeLds<T, DK> L;
  constexpr int NKT = DK / 32;
  extern __shared__ __align__(16) unsigned char smem[];
  const int P = ws.P;
  const int hv = blockIdx.y, b = blockIdx.z;
  const int64_t seq = (int64_t)b * Hv + hv;
  const int lane = threadIdx.x & 63, wave = wave_index();
  const int h = lane >> 5, rr = lane & 31;
  const int n0 = blockIdx.x * 128 + wave * 32;
  const bool active = n0 < DV;  // inactive waves still copy and meet the barriers
  const float* psi = ws.psi + seq * P * DK * DV + n0 + rr;
  f32x16 st[NKT], ps[NKT];
  auto load_psi = [&](int g, f32x16 (&x)[NKT]) {
#pragma unroll
    for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
      for (int i = 0; i < 16; ++i) x[kt][i] = psi[(int64_t)g * DK * DV + (int64_t)(kt * 32 + acc_row(lane, i)) * DV];
  };
  if (active) {
    load_psi(0, st);
    load_psi(1, ps);
  }
  gdr_copy_record(ws.phi + (seq * P + 1) * DK * DK, L::PHI_BYTES, smem, wave, L::PHI_BYTES / 1024);
  for (int g = 1; g < P; ++g) {
    const float* Phi = (const float*)(smem + (size_t)((g - 1) & 1) * L::PHI_BYTES);
    // Phi_g and Psi_g have landed for this wave; the barrier makes that true of every wave and
    // ends every wave's reads of the other buffer.
    pipe_sync<waitcnt_imm(0, 0)>();
    if (g + 1 < P)
      gdr_copy_record(ws.phi + (seq * P + g + 1) * DK * DK, L::PHI_BYTES, smem + (size_t)(g & 1) * L::PHI_BYTES,
                      wave, L::PHI_BYTES / 1024);
    if (active) {
      F sb[NKT][2];
#pragma unroll
      for (int kt = 0; kt < NKT; ++kt) {
        sb[kt][0] = acc_frag<T>(st[kt], 0);
        sb[kt][1] = acc_frag<T>(st[kt], 1);
      }
#pragma unroll
      for (int kt = 0; kt < NKT; ++kt) st[kt] = ps[kt];
      if (g + 1 < P) load_psi(g + 1, ps);
#pragma unroll
      for (int kt = 0; kt < NKT; ++kt) {
        const int i = kt * 32 + rr;
#pragma unroll
        for (int k2 = 0; k2 < NKT; ++k2)
#pragma unroll
          for (int q = 0; q < 2; ++q) {
            const int j = k2 * 32 + 16 * q + 4 * h;
            const f32x4 lo = *(const f32x4*)(Phi + phi_off<DK>(i, j));
            const f32x4 hi = *(const f32x4*)(Phi + phi_off<DK>(i, j + 8));
            F a;
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              a[e] = from_f32<T>(lo[e]);
              a[e + 4] = from_f32<T>(hi[e]);
            }
            mfma_k16(st[kt], a, sb[k2][q]);
          }
      }
    }
  }
  if (!active) return;
  float* Sg = S + seq * DK * DV + n0 + rr;
#pragma unroll
  for (int kt = 0; kt < NKT; ++kt)
#pragma unroll
    for (int i = 0; i < 16; ++i) Sg[(int64_t)(kt * 32 + acc_row(lane, i)) * DV] = st[kt][i];
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
  typedef ChainLds<T, DK, DV> LC;
  static bool once = [] {
    allow_lds_bytes(k_gdr_prep<T, DK, DV>, LP::bytes);
    allow_lds_bytes(k_gdr_chain<T, DK, DV>, LC::bytes);
    allow_lds_bytes(k_gdr_merge<T, DK, DV>, MergeLds<T, DK>::bytes);
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
  const int xblocks = ws.P > 1 ? gdr_xblocks(DK) + gdr_xblocks(DV) : gdr_xblocks(DV);
  k_gdr_chain<T, DK, DV><<<dim3(xblocks, Hv, B * ws.P), gdr::NT, LC::bytes, s>>>(S, ws.gc, Hv, N, ws);
  if (ws.P > 1) {
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    k_gdr_merge<T, DK, DV><<<dim3(gdr_xblocks(DV), Hv, B), gdr::NT, MergeLds<T, DK>::bytes, s>>>(S, Hv, ws);
  }
  record(ev.gdr_scan[1], s);
  return hipGetLastError();
}

// Segments of the two-level scan, from a model of k_gdr_chain fitted on MI355X: one block per
// CU, a chunk step bounded by the record stream of one CU (about 35 GB/s, 1.4 us for a 48 KiB
// record) or by its MFMA chain (about 0.6 us), the records of all offset blocks together by HBM
// (about 4.4 TB/s), and about 3 us per segment in k_gdr_merge. The transition-matrix blocks
// read the same records as the offset blocks of their segment, at about the same time; counting
// their bytes in the HBM term as well made the model choose fewer segments than the measured
// optimum (4 for 256 chunks x 32 heads). P = 1 runs the whole sequence in order. The grid
// dimension B * P stays within 65535.
static void gdr_segments(int NC, int B, int Hv, int dk, int dv, int esize, int& P, int& cps) {
  const double cus = 256.0, merge_us = 3.0, cu_bytes_per_us = 35.0e3, hbm_bytes_per_us = 4.4e6;
  const double seqs = (double)B * Hv;
  const double rec = 64.0 * (2 * dk + dv) * esize;
  const double step_us = std::max(0.6, rec / cu_bytes_per_us);
  const int xk = gdr_xblocks(dk), xv = gdr_xblocks(dv);
  auto cost = [&](int p, int c) {
    const double blocks = seqs * (p > 1 ? (double)p * (xk + xv) - xk : xv);
    const double rounds = std::ceil(blocks / cus);
    const double bytes = seqs * NC * rec * xv;
    const double t = std::max(rounds * c * step_us, bytes / hbm_bytes_per_us);
    return t + (p > 1 ? (p - 1) * merge_us * std::ceil(seqs * xv / cus) : 0.0);
  };
  P = 1;
  cps = NC;
  double best = cost(1, NC);
  const int pmax = std::min(64, std::min(NC / 2, 65535 / B));
  for (int p = 2; p <= pmax; ++p) {
    const int c = (NC + p - 1) / p;
    const int pp = (NC + c - 1) / c;
    const double t = cost(pp, c);
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
  gdr_segments(NC, B, Hv, dk, dv, (int)e, w.P, w.cps);
  w.rec_elems = gdr::C * (2 * dk + dv);
  char* p = (char*)base;
  size_t o = 0;
  w.rec_ = p ? p + o : nullptr;
  o += al((size_t)chunks * w.rec_elems * e);
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
