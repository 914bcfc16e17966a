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

// LDS layout of k_gdr_prep (byte offsets).
template <typename T, int DK, int DV>
struct GdrLds {
  static constexpr int C = gdr::C, P = gdr::PAD;
  static constexpr size_t g = 0;                                   // float[C]  g_t
  static constexpr size_t beta = g + C * 4;                        // float[C]
  static constexpr size_t am = beta + C * 4;                       // float[C][C]    A
  static constexpr size_t tb = am + (size_t)C * C * 4;             // T[C][C+P]      T rounded
  static constexpr size_t vbt = tb + (size_t)C * (C + P) * sizeof(T);     // T[DV][C+P]
  static constexpr size_t kbt = vbt + (size_t)DV * (C + P) * sizeof(T);   // T[DK][C+P]
  static constexpr size_t bytes = kbt + (size_t)DK * (C + P) * sizeof(T);
};

template <typename T, int DK, int DV>
__global__ __launch_bounds__(gdr::NT) void k_gdr_prep(const T* __restrict__ k,
                                                      const T* __restrict__ v,
                                                      const float* __restrict__ alpha,
                                                      const float* __restrict__ beta, int Hk,
                                                      int Hv, int N, GdrWs ws) {
  using namespace gdr;
  typedef GdrLds<T, DK, DV> L;
  extern __shared__ __align__(16) unsigned char smem[];
  float* g = (float*)(smem + L::g);
  float* bet = (float*)(smem + L::beta);
  float* Am = (float*)(smem + L::am);
  T* Tb = (T*)(smem + L::tb);
  T* VbT = (T*)(smem + L::vbt);
  T* KbT = (T*)(smem + L::kbt);
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

  // 1. g_t = prefix sum of log alpha (tokens past N: alpha = 1, beta = 0, k = v = 0).
  if (wave == 0) {
    const bool ok = lane < nval;
    float x = ok ? __logf(fmaxf(alpha[seq * N + t0 + lane], FLT_MIN)) : 0.f;
    const float be = ok ? beta[seq * N + t0 + lane] : 0.f;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const float y = __shfl_up(x, o, WAVE);
      if (lane >= o) x += y;
    }
    g[lane] = x;
    bet[lane] = be;
  }
  __syncthreads();
  const float gC = g[C - 1];

  // 2. Transposed, scaled copies of the chunk: VbT[n][s] = beta_s v_s[n],
  //    KbT[n][s] = beta_s gamma_s k_s[n], and Kt[n][s] = (gamma_C / gamma_s) k_s[n] to HBM.
  T* Kt = ws.kt<T>(seq * NC + c, DK);
  for (int idx = tid; idx < C * (DV / 8); idx += NT) {
    const int s = idx / (DV / 8), n0 = (idx % (DV / 8)) * 8;
    const auto x = s < nval ? frag_load<T>(vc + (int64_t)s * DV + n0) : frag_zero<T>();
    const float bs = bet[s];
#pragma unroll
    for (int e = 0; e < 8; ++e) VbT[(n0 + e) * CP + s] = from_f32<T>(bs * to_f32(x[e]));
  }
  for (int idx = tid; idx < C * (DK / 8); idx += NT) {
    const int s = idx / (DK / 8), n0 = (idx % (DK / 8)) * 8;
    const auto x = s < nval ? frag_load<T>(kc + (int64_t)s * DK + n0) : frag_zero<T>();
    const float a = bet[s] * __expf(g[s]), d = __expf(gC - g[s]);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      KbT[(n0 + e) * CP + s] = from_f32<T>(a * to_f32(x[e]));
      Kt[(n0 + e) * C + s] = from_f32<T>(d * to_f32(x[e]));
    }
  }

  // 3. A[t][s] = beta_t exp(g_t - g_s) k_t.k_s for s < t (K K^T on MFMA, lower tiles only).
  if (wave < 3) {
    const int ti = wave == 0 ? 0 : 1, si = wave == 2 ? 1 : 0;
    const int h = lane >> 5, rr = lane & 31;
    const int ta = ti * 32 + rr, sb = si * 32 + rr;
    f32x16 acc = {};
#pragma unroll
    for (int ks = 0; ks < DK / 16; ++ks) {
      const int ko = ks * 16 + h * 8;
      const auto fa = ta < nval ? frag_load<T>(kc + (int64_t)ta * DK + ko) : frag_zero<T>();
      const auto fb = sb < nval ? frag_load<T>(kc + (int64_t)sb * DK + ko) : frag_zero<T>();
      mfma_k16(acc, fa, fb);
    }
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      const int t = ti * 32 + acc_row(lane, i), s = si * 32 + rr;
      Am[t * C + s] = s < t ? bet[t] * __expf(g[t] - g[s]) * acc[i] : 0.f;
    }
  } else {
    for (int e = lane; e < 32 * 32; e += 64) Am[(e >> 5) * C + 32 + (e & 31)] = 0.f;
  }
  __syncthreads();

  // 4. T = (I + A)^-1 by forward substitution, one column per lane (columns are independent).
  //    Column j of T is zero above row j, so every lane runs the same fully unrolled loops
  //    with its column in registers; the rows of A are read as LDS broadcasts.
  if (wave == 0) {
    const int j = lane;
    float col[C];
#pragma unroll
    for (int i = 0; i < C; ++i) {
      float x = 0.f;
      const float* arow = Am + i * C;
#pragma unroll
      for (int s4 = 0; s4 < i; s4 += 4) {
        const f32x4 a4 = *(const f32x4*)(arow + s4);
#pragma unroll
        for (int u = 0; u < 4; ++u)
          if (s4 + u < i) x -= a4[u] * col[s4 + u];
      }
      col[i] = i < j ? 0.f : (i == j ? 1.f : x);
      Tb[i * CP + j] = from_f32<T>(col[i]);
    }
  }
  __syncthreads();

  // 5. Uv = T (diag(beta) V) and W = T (diag(beta gamma) K), 32x32 tiles over the waves.
  constexpr int NU = (C / 32) * (DV / 32), NW = (C / 32) * (DK / 32);
  T* Uv = ws.uv<T>(seq * NC + c, DV);
  T* W = ws.w<T>(seq * NC + c, DK);
  const int h = lane >> 5, rr = lane & 31;
  for (int q = wave; q < NU + NW; q += NT / 64) {
    const bool isu = q < NU;
    const int qq = isu ? q : q - NU;
    const int nd = isu ? DV / 32 : DK / 32;
    const int ti = qq / nd, ni = qq % nd;
    const T* Bs = isu ? VbT : KbT;
    f32x16 acc = {};
#pragma unroll
    for (int ks = 0; ks < C / 16; ++ks) {
      const int ko = ks * 16 + h * 8;
      mfma_k16(acc, frag_load<T>(Tb + (ti * 32 + rr) * CP + ko),
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
  // entries of this lane's accumulator positions, and Kt rows (A operand of S += Kt U).
  F wf[DK / 16], kf[C / 16];
  T uv[16];
  auto fetch = [&](int c) {
    const int64_t cid = seq * NC + c;
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
    const int64_t cid = seq * NC + c;
    F wnow[DK / 16], know[C / 16];
    T unow[16];
#pragma unroll
    for (int q = 0; q < DK / 16; ++q) wnow[q] = wf[q];
#pragma unroll
    for (int q = 0; q < C / 16; ++q) know[q] = kf[q];
#pragma unroll
    for (int q = 0; q < 16; ++q) unow[q] = uv[q];
    const float gc = ws.gc[cid];
    if (c + 1 < NC) fetch(c + 1);
    // (a) publish the state slice in the call dtype
    if (holds) {
#pragma unroll
      for (int i = 0; i < 16; ++i) Ssh[rr * SP + wave * 32 + acc_row(lane, i)] = from_f32<T>(st[i]);
    }
    __syncthreads();
    // (b) U = Uv - W S for this slice
    if (makes_u) {
      f32x16 acc = {};
#pragma unroll
      for (int ks = 0; ks < DK / 16; ++ks)
        mfma_k16(acc, wnow[ks], *(const F*)(Ssh + rr * SP + ks * 16 + h * 8));
#pragma unroll
      for (int i = 0; i < 16; ++i)
        Ush[rr * UP + wave * 32 + acc_row(lane, i)] = from_f32<T>(to_f32(unow[i]) - acc[i]);
    }
    __syncthreads();
    // (c) S = gamma_C S + Kt U
    if (holds) {
#pragma unroll
      for (int i = 0; i < 16; ++i) st[i] *= gc;
#pragma unroll
      for (int ks = 0; ks < C / 16; ++ks)
        mfma_k16(st, know[ks], *(const F*)(Ush + rr * UP + ks * 16 + h * 8));
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
