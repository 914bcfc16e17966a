// Recurrent adapter (Section 3.1, Eq. 6) on gfx950:
//     M_{-1} = E,   M_l = M_{l-1} + phi(M_{l-1} D_l) U_l   for l = 0 .. L-1,
// followed by the RMSNorm + K/V projection of Section 3.2, Eq. 7 for every layer.
//
// Unlike the embedding adapter, layer l's down projection needs layer l-1's memory, so the
// adapters run as a chain of per-layer kernels:
//   k_down_partial   split-K partial products of M_{l-1} D_l (the T x r output is too small to
//                    fill 256 CUs without splitting the d-long reduction),
//   k_reduce_act     Z_l = phi(sum of the partials) in a fixed order (deterministic),
//   k_up_rec         M_l = M_{l-1} + Z_l U_l: updates the fp32 layer-to-layer state in place,
//                    writes the rounded operand copy for the next layer's down projection, the
//                    memory times gamma_l for the K/V projection and the RMSNorm partial sums.
// The K/V projection of all layers then runs as one launch of the embedding path's kernel.
// The state stays fp32 for every dtype so rounding does not accumulate over the layers.
// bf16 runs with r a multiple of 64 use the pipelined direct-to-LDS engine (k_*_p kernels);
// fp32 runs and other ranks use the register-staged engine.
#include "build_kernels.hpp"
#include "gemm_pipe.hpp"
#include "gemm_tile.hpp"

namespace dv {

template <typename T> struct RecTiles;
template <> struct RecTiles<bf16> { typedef TileCfg<bf16, 128, 128, 2, 2> C; };
template <> struct RecTiles<float> { typedef TileCfg<float, 64, 64, 2, 2> C; };

static inline int rcdiv(int64_t a, int64_t b) { return (int)((a + b - 1) / b); }

// partial[s][t][j] = sum over k in split s of X[t][k] * Dw_l[j][k]
template <class C>
__global__ __launch_bounds__(C::NT) void k_down_partial(const typename C::elem* __restrict__ X,
                                                        const typename C::elem* __restrict__ Dl,
                                                        float* __restrict__ part, int T, int d,
                                                        int r, int kchunk) {
  typedef typename C::elem Tp;
  extern __shared__ __align__(16) unsigned char smem[];
  const int s = blockIdx.z;
  const int k0 = s * kchunk, klen = min(kchunk, d - k0);
  const int n0 = blockIdx.x * C::BN, m0 = blockIdx.y * C::BM;
  f32x16 acc[C::FM][C::FN];
  BRows<Tp> B{Dl + k0, Dl + k0, (int64_t)d, r};
  gemm_nt_mainloop<C>(X + k0, d, T, B, r, klen, m0, n0, (Tp*)smem, acc);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave / C::WGN, wn = wave % C::WGN;
  float* ps = part + (int64_t)s * T * r;
#pragma unroll
  for (int b = 0; b < C::FN; ++b) {
    const int col = n0 + wn * C::WN + b * 32 + (lane & 31);
    if (col >= r) continue;
#pragma unroll
    for (int a = 0; a < C::FM; ++a)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int row = m0 + wm * C::WM + a * 32 + acc_row(lane, i);
        if (row < T) ps[(int64_t)row * r + col] = acc[a][b][i];
      }
  }
}

// Four consecutive elements per thread (n is a multiple of 4: r % 16 == 0); the loop over the
// splits is unrolled so that several splits' loads are in flight at once. The sum runs over the
// splits in order, so the result does not depend on the launch.
template <typename T, int ACT>
__global__ __launch_bounds__(256) void k_reduce_act(const float* __restrict__ part,
                                                    T* __restrict__ Z, int64_t n, int splits) {
  const int64_t i = ((int64_t)blockIdx.x * blockDim.x + threadIdx.x) * 4;
  if (i >= n) return;
  f32x4 x = {0.f, 0.f, 0.f, 0.f};
#pragma unroll 8
  for (int s = 0; s < splits; ++s) x += *(const f32x4*)(part + (int64_t)s * n + i);
#pragma unroll
  for (int u = 0; u < 4; ++u) Z[i + u] = from_f32<T>(ACT == 0 ? silu(x[u]) : gelu(x[u]));
}

// M_l = Min + Z_l U_l. Min is E (layer 0, call dtype) or the fp32 state (it may alias Mst).
template <class C, typename TIn>
__global__ __launch_bounds__(C::NT) void k_up_rec(const TIn* Min, float* Mst,
                                                  typename C::elem* __restrict__ Mop,
                                                  const typename C::elem* __restrict__ Z,
                                                  const typename C::elem* __restrict__ Ul,
                                                  const typename C::elem* __restrict__ gl,
                                                  typename C::elem* __restrict__ Mg,
                                                  float* __restrict__ ssq, int T, int d, int r) {
  typedef typename C::elem Tp;
  extern __shared__ __align__(16) unsigned char smem[];
  const int n0 = blockIdx.x * C::BN, m0 = blockIdx.y * C::BM;
  f32x16 acc[C::FM][C::FN];
  BRows<Tp> B{Ul, Ul, (int64_t)r, d};
  gemm_nt_mainloop<C>(Z, r, T, B, d, r, m0, n0, (Tp*)smem, acc);

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave / C::WGN, wn = wave % C::WGN;
  float part[C::FM][16];
#pragma unroll
  for (int a = 0; a < C::FM; ++a)
#pragma unroll
    for (int i = 0; i < 16; ++i) part[a][i] = 0.f;
#pragma unroll
  for (int b = 0; b < C::FN; ++b) {
    const int col = n0 + wn * C::WN + b * 32 + (lane & 31);
    if (col >= d) continue;
    const float g = to_f32(gl[col]);
#pragma unroll
    for (int a = 0; a < C::FM; ++a)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int row = m0 + wm * C::WM + a * 32 + acc_row(lane, i);
        if (row < T) {
          const int64_t at = (int64_t)row * d + col;
          const float m = acc[a][b][i] + to_f32(Min[at]);
          part[a][i] += m * m;
          Mst[at] = m;
          if (Mop) Mop[at] = from_f32<Tp>(m);
          Mg[at] = from_f32<Tp>(m * g);
        }
      }
  }
#pragma unroll
  for (int a = 0; a < C::FM; ++a)
#pragma unroll
    for (int i = 0; i < 16; ++i) {
      float v = part[a][i];
      v += shfl_xor(v, 1);
      v += shfl_xor(v, 2);
      v += shfl_xor(v, 4);
      v += shfl_xor(v, 8);
      v += shfl_xor(v, 16);
      part[a][i] = v;
    }
  float* red = (float*)smem;  // [WGN][BM]; the main loop ended with a barrier
  if ((lane & 31) == 0) {
#pragma unroll
    for (int a = 0; a < C::FM; ++a)
#pragma unroll
      for (int i = 0; i < 16; ++i) red[wn * C::BM + wm * C::WM + a * 32 + acc_row(lane, i)] = part[a][i];
  }
  __syncthreads();
  for (int rr = threadIdx.x; rr < C::BM; rr += C::NT) {
    const int row = m0 + rr;
    if (row < T) {
      float s = 0.f;
#pragma unroll
      for (int w = 0; w < C::WGN; ++w) s += red[w * C::BM + rr];
      ssq[(int64_t)blockIdx.x * T + row] = s;
    }
  }
}

// ------------------------------------------------------------------ pipelined bf16 kernels

typedef PipeCfg<128, 128, 2, 2> RecP;
// Up-projection epilogue staging: the fp32 tile, rows padded by 4 floats.
constexpr int kRecPitch = RecP::BN + 4;
constexpr int kRecLds = RecP::BM * kRecPitch * 4 > RecP::LDS_BYTES ? RecP::BM * kRecPitch * 4
                                                                   : RecP::LDS_BYTES;

// partial[s][t][j] = sum over k in split s of X[t][k] * Dw_l[j][k]  (one 128x128 tile, one split)
__global__ __launch_bounds__(RecP::NT) void k_down_partial_p(const bf16* __restrict__ X,
                                                             const bf16* __restrict__ Dl,
                                                             float* __restrict__ part, int T, int d,
                                                             int r, int kchunk) {
  typedef RecP C;
  extern __shared__ __align__(16) unsigned char smem[];
  const int s = blockIdx.z;
  const int k0 = s * kchunk, klen = min(kchunk, d - k0);
  const int n0 = blockIdx.x * C::BN, m0 = blockIdx.y * C::BM;
  const int ldb = d * 2;
  // Bases at (first row, first column of the split); the byte ranges end with the matrices,
  // so rows past the end read as zeros.
  BufOperand A{buffer_rsrc(X + (int64_t)m0 * d + k0, (int64_t)(T - m0) * ldb - (int64_t)k0 * 2),
               buffer_rsrc(X, 0), 1 << 30, ldb};
  BufOperand B{buffer_rsrc(Dl + (int64_t)n0 * d + k0, (int64_t)(r - n0) * ldb - (int64_t)k0 * 2),
               buffer_rsrc(Dl, 0), 1 << 30, ldb};
  f32x4 acc[C::FM][C::FN];
  pipe_mainloop<C>(A, B, klen, (bf16*)smem, acc);
  const int lane = threadIdx.x & 63, wave = wave_index();
  const int wm = wave / C::WGN, wn = wave % C::WGN;
  float* ps = part + (int64_t)s * T * r;
#pragma unroll
  for (int a = 0; a < C::FM; ++a) {
    const int row = m0 + wm * C::WM + a * 16 + pipe_row(lane);
    if (row >= T) continue;
#pragma unroll
    for (int b = 0; b < C::FN; ++b) {
      const int col = n0 + wn * C::WN + b * 16 + pipe_col(lane);
      if (col >= r) continue;
      *(f32x4*)(ps + (int64_t)row * r + col) = acc[a][b];
    }
  }
}

// Eight consecutive values of the previous memory as fp32 (bf16 E or the fp32 state).
struct Prev8 {
  f32x4 lo, hi;
};
__device__ __forceinline__ Prev8 load_prev8(const bf16* p) {
  const bf16x8 v = __builtin_bit_cast(bf16x8, *(const u32x4*)p);
  return Prev8{f32x4{(float)v[0], (float)v[1], (float)v[2], (float)v[3]},
               f32x4{(float)v[4], (float)v[5], (float)v[6], (float)v[7]}};
}
__device__ __forceinline__ Prev8 load_prev8(const float* p) {
  return Prev8{*(const f32x4*)p, *(const f32x4*)(p + 4)};
}

// M_l = Min + Z_l U_l for a 128 x 128 tile. Min (E or the fp32 state, which it may alias) is
// fetched before the main loop; the fp32 product goes through padded LDS so that 16 lanes cover
// each 128-column row, and every output moves as whole pieces of a row: the fp32 state, its
// bf16 copy (the next layer's down-projection operand), M * gamma and the row's sum of squares
// over this column tile.
template <typename TIn>
__global__ __launch_bounds__(RecP::NT) void k_up_rec_p(const TIn* Min, float* Mst,
                                                       bf16* __restrict__ Mop,
                                                       const bf16* __restrict__ Z,
                                                       const bf16* __restrict__ Ul,
                                                       const bf16* __restrict__ gl,
                                                       bf16* __restrict__ Mg,
                                                       float* __restrict__ ssq, int T, int d, int r) {
  typedef RecP C;
  extern __shared__ __align__(16) unsigned char smem[];
  const int n0 = blockIdx.x * C::BN, m0 = blockIdx.y * C::BM;
  constexpr int kRows = C::BM / (C::NT / 16);
  const int c8 = (threadIdx.x & 15) * 8;
  const int r16 = threadIdx.x >> 4;
  const bool col_ok = n0 + c8 < d;
  Prev8 prev[kRows];
#pragma unroll
  for (int i = 0; i < kRows; ++i) {
    const int row = m0 + r16 + i * (C::NT / 16);
    prev[i] = (row < T && col_ok) ? load_prev8(Min + (int64_t)row * d + n0 + c8) : Prev8{};
  }
  const int ldb = r * 2;
  BufOperand A{buffer_rsrc(Z + (int64_t)m0 * r, (int64_t)(T - m0) * ldb), buffer_rsrc(Z, 0),
               1 << 30, ldb};
  BufOperand B{buffer_rsrc(Ul + (int64_t)n0 * r, (int64_t)(d - n0) * ldb), buffer_rsrc(Ul, 0),
               1 << 30, ldb};
  f32x4 acc[C::FM][C::FN];
  pipe_mainloop<C>(A, B, r, (bf16*)smem, acc);

  const int lane = threadIdx.x & 63, wave = wave_index();
  const int wm = wave / C::WGN, wn = wave % C::WGN;
  float* tile = (float*)smem;  // the main loop's last LDS read precedes its last barrier
#pragma unroll
  for (int a = 0; a < C::FM; ++a) {
    const int rl = wm * C::WM + a * 16 + pipe_row(lane);
#pragma unroll
    for (int b = 0; b < C::FN; ++b)
      *(f32x4*)(tile + rl * kRecPitch + wn * C::WN + b * 16 + pipe_col(lane)) = acc[a][b];
  }
  __syncthreads();
  bf16x8 g8 = {};
  if (col_ok) g8 = __builtin_bit_cast(bf16x8, *(const u32x4*)(gl + n0 + c8));
#pragma unroll
  for (int i = 0; i < kRows; ++i) {
    const int rr = r16 + i * (C::NT / 16);
    const int row = m0 + rr;
    float ss = 0.f;
    if (row < T && col_ok) {
      const int64_t at = (int64_t)row * d + n0 + c8;
      const f32x4 p0 = *(const f32x4*)(tile + rr * kRecPitch + c8);
      const f32x4 p1 = *(const f32x4*)(tile + rr * kRecPitch + c8 + 4);
      f32x4 m0v, m1v;
      bf16x8 o, mg;
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        m0v[u] = p0[u] + prev[i].lo[u];
        m1v[u] = p1[u] + prev[i].hi[u];
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const float m = u < 4 ? m0v[u] : m1v[u - 4];
        ss += m * m;
        o[u] = (bf16)m;
        mg[u] = (bf16)(m * (float)g8[u]);
      }
      *(f32x4*)(Mst + at) = m0v;
      *(f32x4*)(Mst + at + 4) = m1v;
      if (Mop) *(u32x4*)(Mop + at) = __builtin_bit_cast(u32x4, o);
      __builtin_nontemporal_store(__builtin_bit_cast(u32x4, mg), (u32x4*)(Mg + at));  // read only by the last launch
    }
    ss += shfl_xor(ss, 1);
    ss += shfl_xor(ss, 2);
    ss += shfl_xor(ss, 4);
    ss += shfl_xor(ss, 8);
    if ((threadIdx.x & 15) == 0 && row < T) ssq[(int64_t)blockIdx.x * T + row] = ss;
  }
}

// ------------------------------------------------------------------ host side

static const int kMaxSplits = 16;

// Split of the d-long reduction of the per-layer down projection: enough blocks to fill the
// chip twice (at most kMaxSplits). Returns the chunk length; the split count is cdiv(d, chunk).
template <typename T>
static int rec_kchunk(int T_, int d, int r) {
  typedef typename RecTiles<T>::C C;
  const int64_t blocks = (int64_t)rcdiv(r, C::BN) * rcdiv(T_, C::BM);
  const int ktiles = rcdiv(d, C::BK);
  int s = (int)std::min<int64_t>(kMaxSplits, std::max<int64_t>(1, rcdiv(512, blocks)));
  s = std::min(s, ktiles);
  return rcdiv(ktiles, s) * C::BK;
}

RecLayout recurrent_layout(int64_t T, int d, int L, int r, int dtype) {
  const size_t e = dtype == 1 ? 2 : 4;
  auto al = [](size_t x) { return (x + 255) / 256 * 256; };
  RecLayout w{};
  w.np = dtype == 1 ? rcdiv(d, RecTiles<bf16>::C::BN) : rcdiv(d, RecTiles<float>::C::BN);
  w.kchunk = dtype == 1 ? rec_kchunk<bf16>((int)T, d, r) : rec_kchunk<float>((int)T, d, r);
  w.splits = rcdiv(d, w.kchunk);
  size_t o = 0;
  w.mg = o;      o += al((size_t)L * T * d * e);
  w.ssq = o;     o += al((size_t)L * w.np * T * 4);
  w.state = o;   o += al((size_t)T * d * 4);
  w.op = o;      o += dtype == 1 ? al((size_t)T * d * 2) : 0;
  w.z = o;       o += al((size_t)T * r * e);
  w.part = o;    o += al((size_t)w.splits * T * r * 4);
  w.bytes = o;
  return w;
}

template <typename T>
static hipError_t rec_launch(const void* E, const void* Dw, const void* Uw, const void* gamma,
                             const void* Wk, const void* Wv, void* Kv, void* Vv, int B_, int Nv,
                             int d, int L, int r, int Hkv, int hd, int act, float eps, void* ws,
                             const RecLayout& w, hipStream_t s, const LaunchEvents& ev) {
  typedef typename RecTiles<T>::C C;
  const int T_ = B_ * Nv;
  char* base = (char*)ws;
  T* Mg = (T*)(base + w.mg);
  float* ssq = (float*)(base + w.ssq);
  float* state = (float*)(base + w.state);
  T* op = std::is_same<T, bf16>::value ? (T*)(base + w.op) : nullptr;
  T* Z = (T*)(base + w.z);
  float* part = (float*)(base + w.part);
  const int kchunk = w.kchunk;
  const bool pipelined = std::is_same<T, bf16>::value && r % 64 == 0;
  static bool once = [] {
    (void)hipFuncSetAttribute((const void*)k_up_rec_p<bf16>,
                              hipFuncAttributeMaxDynamicSharedMemorySize, kRecLds);
    (void)hipFuncSetAttribute((const void*)k_up_rec_p<float>,
                              hipFuncAttributeMaxDynamicSharedMemorySize, kRecLds);
    return true;
  }();
  (void)once;
  const int64_t nz = (int64_t)T_ * r;
  dim3 gd(rcdiv(r, C::BN), rcdiv(T_, C::BM), w.splits);
  dim3 gu(rcdiv(d, C::BN), rcdiv(T_, C::BM));
  record(ev.down[0], s);
  for (int l = 0; l < L; ++l) {
    // Operand of this layer's down projection: E for the first layer, then the previous
    // memory (its rounded copy for bf16 runs, the fp32 state itself for fp32 runs).
    const T* X = l == 0 ? (const T*)E : (op ? (const T*)op : (const T*)state);
    if (pipelined)
      k_down_partial_p<<<gd, dim3(RecP::NT), RecP::LDS_BYTES, s>>>(
          (const bf16*)X, (const bf16*)Dw + (int64_t)l * r * d, part, T_, d, r, kchunk);
    else
      k_down_partial<C><<<gd, dim3(C::NT), C::LDS_BYTES, s>>>(X, (const T*)Dw + (int64_t)l * r * d,
                                                              part, T_, d, r, kchunk);
    if (act == 0)
      k_reduce_act<T, 0><<<rcdiv(nz / 4, 256), 256, 0, s>>>(part, Z, nz, w.splits);
    else
      k_reduce_act<T, 1><<<rcdiv(nz / 4, 256), 256, 0, s>>>(part, Z, nz, w.splits);
    const T* Ul = (const T*)Uw + (int64_t)l * d * r;
    const T* gl = (const T*)gamma + (int64_t)l * d;
    T* Mgl = Mg + (int64_t)l * T_ * d;
    float* ssql = ssq + (int64_t)l * w.np * T_;
    if (pipelined && l == 0)
      k_up_rec_p<bf16><<<gu, dim3(RecP::NT), kRecLds, s>>>(
          (const bf16*)E, state, (bf16*)op, (const bf16*)Z, (const bf16*)Ul, (const bf16*)gl,
          (bf16*)Mgl, ssql, T_, d, r);
    else if (pipelined)
      k_up_rec_p<float><<<gu, dim3(RecP::NT), kRecLds, s>>>(
          state, state, (bf16*)op, (const bf16*)Z, (const bf16*)Ul, (const bf16*)gl, (bf16*)Mgl,
          ssql, T_, d, r);
    else if (l == 0)
      k_up_rec<C, T><<<gu, dim3(C::NT), C::LDS_BYTES, s>>>((const T*)E, state, op, Z, Ul, gl, Mgl,
                                                           ssql, T_, d, r);
    else
      k_up_rec<C, float><<<gu, dim3(C::NT), C::LDS_BYTES, s>>>(state, state, op, Z, Ul, gl, Mgl,
                                                               ssql, T_, d, r);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  record(ev.down[1], s);
  return launch_kv_only(Mg, ssq, Wk, Wv, Kv, Vv, B_, Nv, d, Hkv, hd, 0, L, w.np, eps,
                        std::is_same<T, bf16>::value ? 1 : 0, s, ev);
}

hipError_t launch_recurrent(const void* E, const void* Dw, const void* Uw, const void* gamma,
                            const void* Wk, const void* Wv, void* Kv, void* Vv, int B_, int Nv,
                            int d, int L, int r, int Hkv, int hd, int act, float eps, int dtype,
                            void* ws, const RecLayout& w, hipStream_t s, const LaunchEvents& ev) {
  if (dtype == 1)
    return rec_launch<bf16>(E, Dw, Uw, gamma, Wk, Wv, Kv, Vv, B_, Nv, d, L, r, Hkv, hd, act, eps,
                            ws, w, s, ev);
  return rec_launch<float>(E, Dw, Uw, gamma, Wk, Wv, Kv, Vv, B_, Nv, d, L, r, Hkv, hd, act, eps,
                           ws, w, s, ev);
}

}  // namespace dv
