// Visual-memory build and visual K/V projection on gfx950.
//
//   k_down_act   Section 3.1 Eq. 4-5, down half, all layers in one GEMM:
//                Z[l] = phi(E D_l), phi applied to the fp32 accumulators.
//   k_up_norm    Eq. 4-5 up half + residual: M_l = E + Z_l U_l. Writes the
//                memory already multiplied by the RMSNorm weight, rounded to
//                the call dtype, plus fp32 partial sums of M_l^2 per row and
//                column tile (the norm needs the whole row; the partials let
//                the projection finish it without a second pass over M_l).
//   k_kv_proj    Section 3.2 Eq. 7: [Kv | Vv] = (M_l * gamma_l) [Wk | Wv]^T,
//                scaled per row by rsqrt(mean(M_l^2) + eps) in the epilogue
//                (the RMSNorm factor is a per-row scalar, so it commutes with
//                the product), stored head-major [B, Hkv, Nv, hd].
//
// bf16 runs use the pipelined direct-to-LDS engine of gemm_pipe.hpp (k_*_p kernels, one output
// row per lane in the epilogue); fp32 runs, and the bf16 up projection when r is not a multiple
// of 64, use the register-staged engine of gemm_tile.hpp.
#include "build_kernels.hpp"
#include "gemm_pipe.hpp"
#include "gemm_tile.hpp"

#include <atomic>
#include <utility>

namespace dv {

// ---------------------------------------------------------------- tiles

template <typename T> struct BuildTiles;
template <> struct BuildTiles<bf16> {
  typedef TileCfg<bf16, 128, 128, 2, 2> Down;
  typedef TileCfg<bf16, 128, 128, 2, 2> Up;
  typedef TileCfg<bf16, 128, 128, 2, 2> KV;
};
template <> struct BuildTiles<float> {
  typedef TileCfg<float, 64, 64, 2, 2> Down;
  typedef TileCfg<float, 64, 64, 2, 2> Up;
  typedef TileCfg<float, 64, 64, 2, 2> KV;
};

// ---------------------------------------------------------------- K-a

template <class C, int ACT>
__global__ __launch_bounds__(C::NT) void k_down_act(const typename C::elem* __restrict__ E,
                                                    const typename C::elem* __restrict__ Dw,
                                                    typename C::elem* __restrict__ Z, int T,
                                                    int d, int L, int r) {
  typedef typename C::elem Tp;
  extern __shared__ __align__(16) unsigned char smem[];
  Tp* lds = (Tp*)smem;
  const int N = L * r;
  const int n0 = blockIdx.x * C::BN, m0 = blockIdx.y * C::BM;
  f32x16 acc[C::FM][C::FN];
  BRows<Tp> B{Dw, Dw, (int64_t)d, N};
  gemm_nt_mainloop<C>(E, d, T, B, N, d, m0, n0, lds, acc);

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave / C::WGN, wn = wave % C::WGN;
#pragma unroll
  for (int b = 0; b < C::FN; ++b) {
    const int col = n0 + wn * C::WN + b * 32 + (lane & 31);
    if (col >= N) continue;
    const int l = col / r, j = col - l * r;
    Tp* zl = Z + (int64_t)l * T * r + j;
#pragma unroll
    for (int a = 0; a < C::FM; ++a) {
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int row = m0 + wm * C::WM + a * 32 + acc_row(lane, i);
        if (row < T) {
          const float x = acc[a][b][i];
          zl[(int64_t)row * r] = from_f32<Tp>(ACT == 0 ? silu(x) : gelu(x));
        }
      }
    }
  }
}

// ---------------------------------------------------------------- up + residual

template <class C>
__global__ __launch_bounds__(C::NT) void k_up_norm(const typename C::elem* __restrict__ E,
                                                   const typename C::elem* __restrict__ Z,
                                                   const typename C::elem* __restrict__ Uw,
                                                   const typename C::elem* __restrict__ gamma,
                                                   typename C::elem* __restrict__ Mg,
                                                   float* __restrict__ ssq, int T, int d, int r,
                                                   int l0) {
  typedef typename C::elem Tp;
  extern __shared__ __align__(16) unsigned char smem[];
  Tp* lds = (Tp*)smem;
  const int lz = blockIdx.z, l = l0 + lz;
  const int n0 = blockIdx.x * C::BN, m0 = blockIdx.y * C::BM;
  const Tp* Zl = Z + (int64_t)l * T * r;
  const Tp* Ul = Uw + (int64_t)l * d * r;
  f32x16 acc[C::FM][C::FN];
  BRows<Tp> B{Ul, Ul, (int64_t)r, d};
  gemm_nt_mainloop<C>(Zl, r, T, B, d, r, m0, n0, lds, acc);

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave / C::WGN, wn = wave % C::WGN;
  const Tp* gl = gamma + (int64_t)l * d;
  Tp* Ml = Mg + (int64_t)lz * T * d;
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
    for (int a = 0; a < C::FM; ++a) {
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int row = m0 + wm * C::WM + a * 32 + acc_row(lane, i);
        if (row < T) {
          const float m = acc[a][b][i] + to_f32(E[(int64_t)row * d + col]);
          part[a][i] += m * m;
          Ml[(int64_t)row * d + col] = from_f32<Tp>(m * g);
        }
      }
    }
  }
  // Sum the squares over the 32 columns held by each half-wave, then over the
  // WGN waves sharing the rows; one partial per (row, column tile).
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
  const int np = (d + C::BN - 1) / C::BN;
  for (int rr = threadIdx.x; rr < C::BM; rr += C::NT) {
    const int row = m0 + rr;
    if (row < T) {
      float s = 0.f;
#pragma unroll
      for (int w = 0; w < C::WGN; ++w) s += red[w * C::BM + rr];
      ssq[((int64_t)lz * np + blockIdx.x) * T + row] = s;
    }
  }
}

// ---------------------------------------------------------------- K/V projection

template <class C>
__global__ __launch_bounds__(C::NT) void k_kv_proj(const typename C::elem* __restrict__ Mg,
                                                   const float* __restrict__ ssq,
                                                   const typename C::elem* __restrict__ Wk,
                                                   const typename C::elem* __restrict__ Wv,
                                                   typename C::elem* __restrict__ Kv,
                                                   typename C::elem* __restrict__ Vv, int B_,
                                                   int Nv, int d, int Hkv, int hd, int l0,
                                                   int np, float eps) {
  typedef typename C::elem Tp;
  extern __shared__ __align__(16) unsigned char smem[];
  Tp* lds = (Tp*)smem;
  const int T = B_ * Nv, kv = Hkv * hd, N = 2 * kv;
  const int lz = blockIdx.z, l = l0 + lz;
  const int n0 = blockIdx.x * C::BN, m0 = blockIdx.y * C::BM;
  const Tp* Ml = Mg + (int64_t)lz * T * d;
  f32x16 acc[C::FM][C::FN];
  BRows<Tp> Bw{Wk + (int64_t)l * kv * d, Wv + (int64_t)l * kv * d, (int64_t)d, kv};
  gemm_nt_mainloop<C>(Ml, d, T, Bw, N, d, m0, n0, lds, acc);

  // Row scale of the RMSNorm from the partial sums of squares.
  float* rs = (float*)smem;  // [BM]
  for (int rr = threadIdx.x; rr < C::BM; rr += C::NT) {
    const int row = m0 + rr;
    float s = 0.f;
    if (row < T)
      for (int p = 0; p < np; ++p) s += ssq[((int64_t)lz * np + p) * T + row];
    rs[rr] = rsqrtf(s / (float)d + eps);
  }
  __syncthreads();

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave / C::WGN, wn = wave % C::WGN;
  const int64_t head_stride = (int64_t)Nv * hd;
  const int64_t layer_stride = (int64_t)B_ * Hkv * head_stride;
#pragma unroll
  for (int b = 0; b < C::FN; ++b) {
    const int col = n0 + wn * C::WN + b * 32 + (lane & 31);
    if (col >= N) continue;
    Tp* out = col < kv ? Kv : Vv;
    const int o = col < kv ? col : col - kv;
    const int h = o / hd, c = o - h * hd;
    Tp* base = out + (int64_t)l * layer_stride + (int64_t)h * head_stride + c;
#pragma unroll
    for (int a = 0; a < C::FM; ++a) {
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int rl = wm * C::WM + a * 32 + acc_row(lane, i);
        const int row = m0 + rl;
        if (row < T) {
          const int bb = row / Nv, ii = row - bb * Nv;
          base[(int64_t)bb * Hkv * head_stride + (int64_t)ii * hd] = from_f32<Tp>(acc[a][b][i] * rs[rl]);
        }
      }
    }
  }
}


// ---------------------------------------------------------------- bf16 pipelined kernels

typedef PipeCfg<128, 128, 2, 2> DownP;  // two blocks per CU
typedef PipeCfg<192, 128, 4, 2> DownP192;  // 80 KiB of LDS, 96 VGPRs: two blocks per CU
typedef PipeCfg<128, 128, 2, 2> UpP;    // K = r is short; two blocks per CU overlap epilogues
typedef PipeCfg<256, 256, 4, 2> KvP;    // 9216 tiles of 256 x 256 over 32 LLaVA layers
// K/V epilogue staging: per wave 64 rows of 128 bf16, rows padded by 16 B.
constexpr int kKvEpiPitch = KvP::WN * 2 + 16;
constexpr int kKvEpiBytes = KvP::NWAVES * KvP::WM * kKvEpiPitch;
constexpr int kKvRsOffset = KvP::LDS_BYTES > kKvEpiBytes ? KvP::LDS_BYTES : kKvEpiBytes;
constexpr int kKvLdsBytes = kKvRsOffset + KvP::BM * 4;  // + row scales

// Output tile (row tile mt, column tile nt) of a block when the tiles of one XCD should form
// compact supertiles. The dispatcher deals consecutive workgroup ids out to the 8 XCDs in turn, so
// in launch order (column tile fastest) every XCD touches every row tile and the blocks that share
// an operand tile sit on different L2s. Here the ids of each XCD (id % 8) are renumbered to be
// consecutive, XCD x taking the x-th eighth of the tile sequence, and the sequence walks bands of
// sh row tiles, each band in sh x sw supertiles (row within the supertile slowest). The blocks an
// XCD holds at once then share a few row tiles and a few column tiles of the two operands. Ids past
// the last multiple of 8 keep their place; sh == 0 keeps launch order. Grid x = column tiles,
// y = row tiles; z (layers) is left to the caller.
struct Tile2 {
  int mt, nt;
};
__device__ __forceinline__ Tile2 supertile_order(int sh, int sw) {
  if (sh == 0) return Tile2{(int)blockIdx.y, (int)blockIdx.x};
  const int gx = gridDim.x, gy = gridDim.y;
  const int id = blockIdx.x + gx * blockIdx.y;
  const int per = gx * gy / 8, full = per * 8;
  const int q = id < full ? (id % 8) * per + id / 8 : id;
  const int band = q / (sh * gx);
  const int h = min(sh, gy - band * sh);
  const int in = q - band * sh * gx;
  const int cs = in / (h * sw);
  const int w = min(sw, gx - cs * sw);
  const int j = in - cs * h * sw;
  return Tile2{band * sh + j / w, cs * sw + j % w};
}

template <typename F>
__device__ __forceinline__ void store4_bf16(bf16* p, float a, float b, float c, float d, F f) {
  bf16x4 v = {(bf16)f(a), (bf16)f(b), (bf16)f(c), (bf16)f(d)};
  *(u32x2*)p = __builtin_bit_cast(u32x2, v);
}

__device__ __forceinline__ void load4_bf16(const bf16* p, float (&x)[4]) {
  bf16x4 v = __builtin_bit_cast(bf16x4, *(const u32x2*)p);
#pragma unroll
  for (int e = 0; e < 4; ++e) x[e] = (float)v[e];
}

template <class C, int ACT>
__global__ __launch_bounds__(C::NT) void k_down_act_p(const bf16* __restrict__ E,
                                                      const bf16* __restrict__ Dw,
                                                      bf16* __restrict__ Z, int T, int d, int L,
                                                      int r, int sh, int sw) {
  extern __shared__ __align__(16) unsigned char smem[];
  const int N = L * r;
  const Tile2 tile = supertile_order(sh, sw);
  const int n0 = tile.nt * C::BN, m0 = tile.mt * C::BM;
  const int ldb = d * 2;
  BufOperand A{buffer_rsrc(E + (int64_t)m0 * d, (int64_t)(T - m0) * ldb),
               buffer_rsrc(E, 0), 1 << 30, ldb};
  BufOperand B{buffer_rsrc(Dw + (int64_t)n0 * d, (int64_t)(N - n0) * ldb),
               buffer_rsrc(Dw, 0), 1 << 30, ldb};
  f32x4 acc[C::FM][C::FN];
  pipe_mainloop<C>(A, B, d, (bf16*)smem, acc);

  const int lane = threadIdx.x & 63, wave = wave_index();
  const int wm = wave / C::WGN, wn = wave % C::WGN;
#pragma unroll
  for (int a = 0; a < C::FM; ++a) {
    const int row = m0 + wm * C::WM + a * 16 + pipe_row(lane);
    if (row >= T) continue;
#pragma unroll
    for (int b = 0; b < C::FN; ++b) {
      const int n = n0 + wn * C::WN + b * 16 + pipe_col(lane);  // r % 16 == 0: one layer
      if (n >= N) continue;
      const int l = n / r, j = n - l * r;
      const f32x4& v = acc[a][b];
      store4_bf16(Z + ((int64_t)l * T + row) * r + j, v[0], v[1], v[2], v[3],
                  [](float x) { return ACT == 0 ? silu(x) : gelu(x); });
    }
  }
}

// Up-projection epilogue scratch past the two stages: per wave a 16 x 64 bf16 transpose buffer
// (rows padded by 16 bytes), then the per-row sums of squares of the two column halves.
template <class C>
struct UpLds {
  static constexpr int SCR_PITCH = C::WN + 8;  // bf16 elements
  static constexpr int SCR = C::LDS_BYTES;
  static constexpr int SS = SCR + C::NWAVES * 16 * SCR_PITCH * 2;
  static constexpr int BYTES = SS + C::WGN * C::BM * 4;
};


// One 128 x 128 tile of M_l * gamma_l for kUpLayers consecutive layers through one pipeline
// (the next layer's first operand tiles load while a layer's epilogue runs). The epilogue works
// on the accumulators in place: lane l holds row l % 16 of each 16-row fragment and four
// consecutive columns, E and gamma are fetched in that layout, the per-row sum of squares of fp32
// M is a shuffle over the four lanes of a row plus one LDS exchange between the two waves of a
// row band, and each wave turns its bf16 rows around through a 2 KiB LDS buffer so that they
// leave as whole 128-byte lines.
template <class C>
__global__ __launch_bounds__(C::NT) void k_up_norm_p(const bf16* __restrict__ E,
                                                       const bf16* __restrict__ Z,
                                                       const bf16* __restrict__ Uw,
                                                       const bf16* __restrict__ gamma,
                                                       bf16* __restrict__ Mg,
                                                       float* __restrict__ ssq, int T, int d,
                                                       int r, int l0, int nl, int lpb, int sh,
                                                       int sw) {
  static_assert(C::WGN == 2 && C::WN == 64, "epilogue assumes two 64-column wave halves");
  extern __shared__ __align__(16) unsigned char smem[];
  const Tile2 tile = supertile_order(sh, sw);
  const int n0 = tile.nt * C::BN, m0 = tile.mt * C::BM;
  const int lz0 = blockIdx.z * lpb, nrun = min(nl - lz0, lpb);
  const int ldb = r * 2;
  const int lane = threadIdx.x & 63, wave = wave_index();
  const int wm = wave / C::WGN, wn = wave % C::WGN;
  const int row0 = m0 + wm * C::WM + pipe_row(lane);       // + a * 16
  const int col0 = n0 + wn * C::WN + pipe_col(lane);       // + b * 16
  const bool cols_ok = n0 + wn * C::WN < d;  // d % 64 == 0: a wave's 64 columns are all in or out
  // E in the accumulator layout, fetched once for every layer of the block.
  u32x2 e4[C::FM][C::FN];
#pragma unroll
  for (int a = 0; a < C::FM; ++a)
#pragma unroll
    for (int b = 0; b < C::FN; ++b)
      e4[a][b] = (cols_ok && row0 + a * 16 < T)
                     ? *(const u32x2*)(E + (int64_t)(row0 + a * 16) * d + col0 + b * 16)
                     : u32x2{};
  auto load_gamma = [&](int lz, u32x2 (&g)[C::FN]) {
#pragma unroll
    for (int b = 0; b < C::FN; ++b)
      g[b] = cols_ok ? *(const u32x2*)(gamma + (int64_t)(l0 + lz) * d + col0 + b * 16) : u32x2{};
  };
  u32x2 g4[C::FN];
  load_gamma(lz0, g4);
  constexpr int kUpScrPitch = UpLds<C>::SCR_PITCH;
  bf16* scr = (bf16*)(smem + UpLds<C>::SCR) + wave * 16 * kUpScrPitch;
  float* ssx = (float*)(smem + UpLds<C>::SS);
  const int np = (d + C::BN - 1) / C::BN;

  auto operands = [&](int run, BufOperand& A, BufOperand& B) {
    const int l = l0 + lz0 + run;
    const bf16* Zl = Z + (int64_t)l * T * r;
    const bf16* Ul = Uw + (int64_t)l * d * r;
    A = BufOperand{buffer_rsrc(Zl + (int64_t)m0 * r, (int64_t)(T - m0) * ldb), buffer_rsrc(Zl, 0),
                   1 << 30, ldb};
    B = BufOperand{buffer_rsrc(Ul + (int64_t)n0 * r, (int64_t)(d - n0) * ldb), buffer_rsrc(Ul, 0),
                   1 << 30, ldb};
  };
  auto epilogue = [&](int run, f32x4 (&acc)[C::FM][C::FN]) {
    const int lz = lz0 + run;
    bf16* Ml = Mg + (int64_t)lz * T * d;
    float ssr[C::FM];
#pragma unroll
    for (int a = 0; a < C::FM; ++a) {
      float ss = 0.f;
#pragma unroll
      for (int b = 0; b < C::FN; ++b) {
        const bf16x4 e = __builtin_bit_cast(bf16x4, e4[a][b]);
        const bf16x4 g = __builtin_bit_cast(bf16x4, g4[b]);
        bf16x4 o;
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const float m = acc[a][b][u] + (float)e[u];
          ss += m * m;
          o[u] = (bf16)(m * (float)g[u]);
        }
        *(u32x2*)(scr + pipe_row(lane) * kUpScrPitch + b * 16 + pipe_col(lane)) =
            __builtin_bit_cast(u32x2, o);
      }
      ss += shfl_xor(ss, 16);
      ss += shfl_xor(ss, 32);
      ssr[a] = ss;
      // The buffer is this wave's own: LDS serves a wave's accesses in order, so a wave-level
      // fence is all the read-back needs.
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int rr = h * 8 + (lane >> 3);
        const u32x4 v = *(const u32x4*)(scr + rr * kUpScrPitch + (lane & 7) * 8);
        const int row = m0 + wm * C::WM + a * 16 + rr;
        // Streaming store: M * gamma of all layers (0.6 GB at LLaVA-7B shapes) is read only by
        // the projection launch; through the caches the stores ran at about 1.8 TB/s.
        if (cols_ok && row < T)
          __builtin_nontemporal_store(
              v, (u32x4*)(Ml + (int64_t)row * d + n0 + wn * C::WN + (lane & 7) * 8));
      }
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    }
    if (run + 1 < nrun) load_gamma(lz + 1, g4);
    // Row sums of the two column halves meet in LDS. The previous layer's exchange was read
    // before at least one barrier of this layer's main loop.
    if (lane < 16) {
#pragma unroll
      for (int a = 0; a < C::FM; ++a) ssx[wn * C::BM + wm * C::WM + a * 16 + lane] = ssr[a];
    }
    pipe_sync<waitcnt_imm(63, 0)>();  // LDS writes done; the stores stay in flight
    if (threadIdx.x < C::BM) {
      const int row = m0 + threadIdx.x;
      if (row < T)
        ssq[((int64_t)lz * np + tile.nt) * T + row] = ssx[threadIdx.x] + ssx[C::BM + threadIdx.x];
    }
  };
  pipe_runs<C>(nrun, r, (bf16*)smem, operands, epilogue);
}

// ------------------------------------------------------------------ up projection, Z resident
//
// For a large rank (r = 512) and many token tiles the up projection can run the other way
// round: a block takes one 128-row tile of one layer and walks every 128-column tile of d, and
// each of its four waves (64 x 64 of the tile, one per SIMD) holds its 64 rows of Z_l for the
// whole layer in registers (r / 2 of them, mostly accumulation registers, which the MFMAs read
// directly). Only U streams through LDS, in a four-deep ring per wave that no other wave reads,
// so the main loop has no barrier, and every wave sees whole rows of M: the block writes the
// full-row sum of squares (one partial per row instead of one per column tile). E comes through
// the wave's LDS as whole 128-byte rows and is read back in the accumulator layout; the same
// buffer then turns M * gamma around for the stores.
// Every load and store of the loop is a buffer instruction issued unconditionally (rows and
// columns outside the tensors take out-of-range offsets: loads return zeros, stores are dropped)
// and the LDS traffic is inline assembly, so the number of memory instructions a wave has in
// flight is the same on every path and the waits below count them exactly.
template <int I, int N, class F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (I < N) {
    f(std::integral_constant<int, I>{});
    static_for<I + 1, N>(f);
  }
}

namespace upz {
constexpr int BM = 128, BN = 128, NW = 4, WM = 64, WN = 64, FM = WM / 16, FN = WN / 16;
constexpr int D = 4;                          // U tiles in flight per wave
constexpr int TILE = WN * 128;                // one wave's U tile: 64 columns x 64 k (8 KiB)
constexpr int RING = D * TILE;
constexpr int EBUF = WM * WN * 2;             // one wave's E tile (8 KiB), then the turnaround
constexpr int SCR_PITCH = WN + 8;             // bf16 per row of the store turnaround
constexpr int WAVE_LDS = RING + EBUF;
constexpr int LDS_BYTES = NW * WAVE_LDS;      // 160 KiB; the row-sum exchange reuses it
constexpr int DMA = TILE / 1024;              // 1 KiB load instructions per U tile
// Counted loads per column tile: E's. Only instructions the compiler cannot move are counted
// (loads into LDS and stores have side effects and keep their order); gamma's loads write
// registers, may be moved (the compiler waits for them itself), and an uncounted instruction only
// makes a wait stricter.
constexpr int G = EBUF / 1024;
constexpr int S = 2 * FM;                     // M * gamma stores per column tile
constexpr uint32_t OOR = 0x80000000u;         // past every buffer's range
constexpr int CPOL_NT = 2;                    // non-temporal: M * gamma is read by the next launch
static_assert(DMA * (D - 1) + S + G <= 63, "vmcnt counts every instruction in flight");
static_assert(16 * SCR_PITCH * 2 <= EBUF, "the turnaround fits in the E buffer");

template <int OFF>
__device__ __forceinline__ u32x4 lds_read_b128(uint32_t addr) {
  static_assert(OFF >= 0 && OFF < 65536, "16-bit LDS offset");
  u32x4 r;
  asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(r) : "v"(addr), "n"(OFF));
  return r;
}
template <int OFF>
__device__ __forceinline__ u32x2 lds_read_b64(uint32_t addr) {
  static_assert(OFF >= 0 && OFF < 65536, "16-bit LDS offset");
  u32x2 r;
  asm volatile("ds_read_b64 %0, %1 offset:%2" : "=v"(r) : "v"(addr), "n"(OFF));
  return r;
}
__device__ __forceinline__ void lds_write_b64(uint32_t addr, u32x2 v) {
  asm volatile("ds_write_b64 %0, %1" ::"v"(addr), "v"(v) : "memory");
}
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
}
// Wait for the LDS reads in flight and tie their results to this point.
template <class V, int N>
__device__ __forceinline__ void lds_wait(V (&v)[N]) {
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
#pragma unroll
  for (int i = 0; i < N; ++i) asm volatile("" : "+v"(v[i]));
}
// Vector-memory wait for the U tile after tile kt of a column tile. In flight, oldest first:
// that tile, the D - 1 tiles after it, and, for kt <= D - 2, the previous column tile's stores
// and this column tile's E loads, issued after that tile's loads.
template <int KT, bool FIRST>
__device__ __forceinline__ void wait_next() {
  constexpr int n = DMA * (D - 1) + (KT <= D - 2 ? G + (FIRST ? 0 : S) : 0);
  __builtin_amdgcn_s_waitcnt(waitcnt_imm(n, 15));
  asm volatile("" ::: "memory");
}
}  // namespace upz

template <int R>
__global__ __launch_bounds__(upz::NW * 64, 1) void k_up_norm_zr(
    const bf16* __restrict__ E, const bf16* __restrict__ Z, const bf16* __restrict__ Uw,
    const bf16* __restrict__ gamma, bf16* __restrict__ Mg, float* __restrict__ ssq, int T, int d,
    int l0, int nl) {
  using namespace upz;
  constexpr int KS = R / 32;   // 32-deep MFMA steps per column tile
  constexpr int NKT = R / 64;  // 64-deep U tiles per column tile
  static_assert(NKT % D == 0 && NKT >= D, "the ring slot of a tile is its index mod D");
  extern __shared__ __align__(16) unsigned char smem[];
  const int lane = threadIdx.x & 63, wave = wave_index();
  const int wm = wave >> 1, wn = wave & 1;
  // Layer-major block order: the blocks an XCD holds at once share a layer and so its U.
  const int n_rt = (T + BM - 1) / BM;
  const int lz = blockIdx.x / n_rt, m0 = (blockIdx.x - lz * n_rt) * BM;
  const int l = l0 + lz;
  const int ncol = (d + BN - 1) / BN;
  const int row0 = m0 + wm * WM + (lane & 15);  // + 16 a: this lane's rows
  const int kq = 8 * (lane >> 4);                 // this lane's k offset within a 32-deep step

  // Z_l rows of this wave, in the B-operand layout of the MFMAs (swapped, as in the GEMMs).
  const __amdgpu_buffer_rsrc_t rz = buffer_rsrc(Z + (int64_t)l * T * R, (int64_t)T * R * 2);
  bf16x8 zf[KS][FM];
#pragma unroll
  for (int s = 0; s < KS; ++s)
#pragma unroll
    for (int a = 0; a < FM; ++a)
      zf[s][a] = __builtin_bit_cast(
          bf16x8, __builtin_amdgcn_raw_buffer_load_b128(
                      rz, ((row0 + 16 * a) * R + 32 * s + kq) * 2, 0, 0));
  __builtin_amdgcn_s_waitcnt(waitcnt_imm(0, 15));  // Z is complete before the streams start

  // U tile p of the stream (column tile p / NKT, K tile p % NKT) of this wave: rows
  // j*128 + wn*64 + 0..63 of U_l (the output columns), bytes 128*kt .. +127 of each row, into
  // ring slot p % D with the GEMM pipeline's swizzled layout. E tiles use the same layout.
  const __amdgpu_buffer_rsrc_t ru = buffer_rsrc(Uw + (int64_t)l * d * R, (int64_t)d * R * 2);
  const __amdgpu_buffer_rsrc_t re = buffer_rsrc(E, (int64_t)T * d * 2);
  const __amdgpu_buffer_rsrc_t rg = buffer_rsrc(gamma + (int64_t)l * d, (int64_t)d * 2);
  const __amdgpu_buffer_rsrc_t rm = buffer_rsrc(Mg + (int64_t)lz * T * d, (int64_t)T * d * 2);
  const int ua0 = pipe_lane_offset(R * 2, 0), ua1 = pipe_lane_offset(R * 2, 1);
  const int ea0 = pipe_lane_offset(d * 2, 0), ea1 = pipe_lane_offset(d * 2, 1);
  unsigned char* ring = smem + wave * WAVE_LDS;
  unsigned char* ebuf = ring + RING;
  auto issue_u = [&](int j, int kt, int slot) {
    const bool in = j < ncol;
    const int sbase = (j * BN + wn * WN) * R * 2 + kt * 128;
#pragma unroll
    for (int blk = 0; blk < DMA; ++blk)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          ru, (lds_void*)(ring + slot * TILE + blk * 1024), 16, (blk & 1) ? ua1 : ua0,
          in ? sbase + blk * 8 * R * 2 : (int)OOR, 0, 0);
  };
  // E rows m0 + wm*64 + 0..63, columns c0 .. c0 + 63 (128 bytes of each row), and gamma.
  u32x2 g4[FN];
  auto issue_eg = [&](int j) {
    const int c0 = j * BN + wn * WN;
    const bool in = c0 < d;  // d % 64 == 0: the wave's 64 columns are all in or out
#pragma unroll
    for (int blk = 0; blk < EBUF / 1024; ++blk) {
      const int r8 = m0 + wm * WM + blk * 8;  // rows past T read zeros (past the range)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(re, (lds_void*)(ebuf + blk * 1024), 16,
                                               (blk & 1) ? ea1 : ea0,
                                               in ? (r8 * d + c0) * 2 : (int)OOR, 0, 0);
    }
#pragma unroll
    for (int b = 0; b < FN; ++b)
      g4[b] = __builtin_amdgcn_raw_buffer_load_b64(
          rg, in ? (c0 + 16 * b + 4 * (lane >> 4)) * 2 : OOR, 0, 0);
  };
  // Fragment b of K step s2 of a U tile: row b*16 + lane%16, 16-byte chunk 4*s2 + lane/16, XOR
  // key (row / 2) % 8 = (lane % 16) / 2. E in the accumulator layout: row a*16 + lane%16, bytes
  // 8*(lane/16) + 32 b of the row, i.e. chunk 2b + lane/32 at byte 8*((lane/16) % 2).
  const uint32_t ring_addr = lds_addr(ring), e_addr = lds_addr(ebuf);
  const int key = (lane & 15) >> 1;
  uint32_t fo[2];
#pragma unroll
  for (int s2 = 0; s2 < 2; ++s2)
    fo[s2] = ring_addr + (lane & 15) * 128 + (((4 * s2 + (lane >> 4)) ^ key) << 4);
  uint32_t eo[FN];
#pragma unroll
  for (int b = 0; b < FN; ++b)
    eo[b] = e_addr + (lane & 15) * 128 + (((2 * b + (lane >> 5)) ^ key) << 4) + 8 * ((lane >> 4) & 1);
  const uint32_t scr_w = e_addr + ((lane & 15) * SCR_PITCH + 4 * (lane >> 4)) * 2;
  const uint32_t scr_r = e_addr + ((lane >> 3) * SCR_PITCH + (lane & 7) * 8) * 2;

  auto read_frags = [&](auto slotc, u32x4 (&f)[2][FN]) {
    constexpr int slot = decltype(slotc)::value;
#pragma unroll
    for (int s2 = 0; s2 < 2; ++s2) {
      f[s2][0] = upz::lds_read_b128<slot * TILE + 0 * 2048>(fo[s2]);
      f[s2][1] = upz::lds_read_b128<slot * TILE + 1 * 2048>(fo[s2]);
      f[s2][2] = upz::lds_read_b128<slot * TILE + 2 * 2048>(fo[s2]);
      f[s2][3] = upz::lds_read_b128<slot * TILE + 3 * 2048>(fo[s2]);
    }
  };

#pragma unroll
  for (int kt = 0; kt < D; ++kt) issue_u(0, kt, kt);
  issue_eg(0);
  __builtin_amdgcn_s_waitcnt(waitcnt_imm(DMA * (D - 1) + G, 15));  // U tile 0 landed
  asm volatile("" ::: "memory");
  u32x4 fr[2][2][FN];  // fragments of the current and the next U tile
  read_frags(std::integral_constant<int, 0>{}, fr[0]);
  float ss[FM] = {0.f, 0.f, 0.f, 0.f};
  for (int j = 0; j < ncol; ++j) {
    const int c0 = j * BN + wn * WN;  // this wave's first column
    const bool cols_ok = c0 < d;
    if (j > 0) issue_eg(j);
    f32x4 acc[FM][FN];
#pragma unroll
    for (int a = 0; a < FM; ++a)
#pragma unroll
      for (int b = 0; b < FN; ++b) acc[a][b] = f32x4{};
    const bool first = j == 0;
    static_for<0, NKT>([&](auto ktc) {
      constexpr int kt = decltype(ktc)::value, slot = kt % D, cur = kt & 1;
      upz::lds_wait(fr[cur][0]);
      upz::lds_wait(fr[cur][1]);
      // This tile's slot is read: refill it with the tile D ahead in the stream.
      constexpr int nxt = kt + D;
      issue_u(nxt < NKT ? j : j + 1, nxt % NKT, slot);
      // The next tile (the next column tile's first one after the last) lands, then its
      // fragments are read while this tile's MFMAs run.
      if (first) upz::wait_next<kt, true>();
      else upz::wait_next<kt, false>();
      read_frags(std::integral_constant<int, (kt + 1) % D>{}, fr[cur ^ 1]);
#pragma unroll
      for (int s2 = 0; s2 < 2; ++s2)
#pragma unroll
        for (int a = 0; a < FM; ++a)
#pragma unroll
          for (int b = 0; b < FN; ++b)
            acc[a][b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                __builtin_bit_cast(bf16x8, fr[cur][s2][b]), zf[2 * kt + s2][a], acc[a][b], 0, 0,
                0);
    });
    static_assert(NKT % 2 == 0, "the next column tile's first fragments sit in fr[0]");

    // Epilogue: M = acc + E, the row sums of squares of fp32 M, M * gamma rounded to bf16 and
    // turned around through the E buffer so that every store writes 16-byte pieces of rows.
    // E of this column tile landed before the last wait above (it was issued before the U tile
    // waited for there).
#pragma unroll
    for (int a = 0; a < FM; ++a) {
      u32x2 e4[FN];
      e4[0] = upz::lds_read_b64<0>(eo[0] + a * 16 * 128);
      e4[1] = upz::lds_read_b64<0>(eo[1] + a * 16 * 128);
      e4[2] = upz::lds_read_b64<0>(eo[2] + a * 16 * 128);
      e4[3] = upz::lds_read_b64<0>(eo[3] + a * 16 * 128);
      upz::lds_wait(e4);
#pragma unroll
      for (int b = 0; b < FN; ++b) {
        const bf16x4 e = __builtin_bit_cast(bf16x4, e4[b]);
        const bf16x4 g = __builtin_bit_cast(bf16x4, g4[b]);
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const float m = acc[a][b][u] + (float)e[u];
          ss[a] += m * m;
          acc[a][b][u] = m * (float)g[u];
        }
      }
    }
#pragma unroll
    for (int a = 0; a < FM; ++a) {
#pragma unroll
      for (int b = 0; b < FN; ++b) {
        bf16x4 o;
#pragma unroll
        for (int u = 0; u < 4; ++u) o[u] = (bf16)acc[a][b][u];
        upz::lds_write_b64(scr_w + b * 32, __builtin_bit_cast(u32x2, o));
      }
      u32x4 v[2];
      v[0] = upz::lds_read_b128<0>(scr_r);
      v[1] = upz::lds_read_b128<8 * SCR_PITCH * 2>(scr_r);
      upz::lds_wait(v);
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int row = m0 + wm * WM + a * 16 + h * 8 + (lane >> 3);
        __builtin_amdgcn_raw_buffer_store_b128(
            v[h], rm, (cols_ok && row < T) ? (row * d + c0 + (lane & 7) * 8) * 2 : OOR, 0,
            CPOL_NT);
      }
    }
  }
  // Row sums of squares: the four lanes of a row, then the two column halves through LDS.
  __builtin_amdgcn_s_waitcnt(waitcnt_imm(0, 0));  // nothing of the streams is in flight
  __syncthreads();
  float* ssx = (float*)smem;
#pragma unroll
  for (int a = 0; a < FM; ++a) {
    float s = ss[a];
    s += shfl_xor(s, 16);
    s += shfl_xor(s, 32);
    if (lane < 16) ssx[wn * BM + wm * WM + a * 16 + lane] = s;
  }
  __syncthreads();
  if (threadIdx.x < BM && m0 + (int)threadIdx.x < T)
    ssq[(int64_t)lz * T + m0 + threadIdx.x] = ssx[threadIdx.x] + ssx[BM + threadIdx.x];
}

// Backbone epilogue arguments as the kernels see them (see KvEpiArgs).
template <typename T>
struct KvEpi {
  const T* kb;
  const T* vb;
  const T* kn;
  float kn_eps;
  const float* rope;
};

template <typename T>
static KvEpi<T> epi_dev(const KvEpiArgs* a) {
  if (!a) return KvEpi<T>{nullptr, nullptr, nullptr, 0.f, nullptr};
  return KvEpi<T>{(const T*)a->k_bias, (const T*)a->v_bias, (const T*)a->k_norm, a->k_norm_eps,
                  a->rope};
}

__device__ __forceinline__ void unpack8(const u32x4 v, float (&x)[8]) {
  const bf16x8 b = __builtin_bit_cast(bf16x8, v);
#pragma unroll
  for (int e = 0; e < 8; ++e) x[e] = (float)b[e];
}

__device__ __forceinline__ u32x4 pack8(const float (&x)[8]) {
  bf16x8 b;
#pragma unroll
  for (int e = 0; e < 8; ++e) b[e] = (bf16)x[e];
  return __builtin_bit_cast(u32x4, b);
}

// Tile of a K/V projection block: layer lz (within the call), row tile mt, column tile nt.
// The dispatcher deals consecutive launch ids out to the 8 XCDs in turn. In launch order (column
// tile fastest) an XCD holds every row tile of a few column tiles: each weight tile stays on one
// XCD and each row tile of M * gamma is fetched by every XCD. With rows_by_xcd the row tiles are
// dealt out instead (tiles x, x + 8, ... to one XCD, column tile fastest within it): each M * gamma
// tile stays on one XCD and the weights are fetched by every XCD. The host picks the order that
// fetches fewer bytes from beyond the L2s.
struct KvTile {
  int lz, mt, nt;
};
__device__ __forceinline__ KvTile kv_tile(int rows_by_xcd) {
  if (!rows_by_xcd) return KvTile{(int)blockIdx.z, (int)blockIdx.y, (int)blockIdx.x};
  const int gx = gridDim.x, gy = gridDim.y;
  const int r = blockIdx.x + gx * blockIdx.y;  // launch order within the layer
  const int full = (gy / 8) * 8 * gx;            // row tiles that fill all 8 XCDs
  int mt, nt;
  if (r < full) {
    const int slot = r / 8;
    nt = slot % gx;
    mt = (slot / gx) * 8 + r % 8;
  } else {
    nt = (r - full) % gx;
    mt = (gy / 8) * 8 + (r - full) / gx;
  }
  return KvTile{(int)blockIdx.z, mt, nt};
}

// EPI adds the backbone epilogue: the bias joins the scaled product before it is rounded to
// the call dtype (as the backbone's projection would), then the staged head rows of K get the
// per-head RMSNorm and the rotary embedding (the partner half of a head is read from the
// staging buffer) before their single final rounding.
template <bool EPI>
__global__ __launch_bounds__(KvP::NT) void k_kv_proj_p(const bf16* __restrict__ Mg,
                                                       const float* __restrict__ ssq,
                                                       const bf16* __restrict__ Wk,
                                                       const bf16* __restrict__ Wv,
                                                       bf16* __restrict__ Kv, bf16* __restrict__ Vv,
                                                       int B_, int Nv, int d, int Hkv, int hd,
                                                       int l0, int np, float eps, KvEpi<bf16> epi,
                                                       int rows_by_xcd) {
  typedef KvP C;
  extern __shared__ __align__(16) unsigned char smem[];
  const int T = B_ * Nv, kv = Hkv * hd, N = 2 * kv;
  const KvTile tile = kv_tile(rows_by_xcd);
  const int lz = tile.lz, l = l0 + lz;
  const int n0 = tile.nt * C::BN, m0 = tile.mt * C::BM;
  const bf16* Ml = Mg + (int64_t)lz * T * d;
  const bf16* Wkl = Wk + (int64_t)l * kv * d;
  const bf16* Wvl = Wv + (int64_t)l * kv * d;
  const int ldb = d * 2;
  BufOperand A{buffer_rsrc(Ml + (int64_t)m0 * d, (int64_t)(T - m0) * ldb), buffer_rsrc(Ml, 0),
               1 << 30, ldb};
  BufOperand B;
  if (n0 < kv) {
    B = BufOperand{buffer_rsrc(Wkl + (int64_t)n0 * d, (int64_t)(kv - n0) * ldb),
                   buffer_rsrc(Wvl, (int64_t)kv * ldb), kv - n0, ldb};
  } else {
    B = BufOperand{buffer_rsrc(Wvl + (int64_t)(n0 - kv) * d, (int64_t)(N - n0) * ldb),
                   buffer_rsrc(Wvl, 0), 1 << 30, ldb};
  }
  // RMSNorm row scales of this block's rows from the partial sums of squares, two threads per
  // row. The first 64 partials of each row are requested before the operand tiles (so their
  // latency hides behind the pipeline's first wait) and summed, in a fixed order, after the
  // main loop; the scales go to the LDS bytes above the two pipeline stages.
  float* rs_lds = (float*)(smem + kKvRsOffset);
  const int rs_r = threadIdx.x >> 1, rs_half = threadIdx.x & 1;
  const int rs_row = m0 + rs_r;
  const float* rs_src = ssq + (int64_t)lz * np * T + rs_row;
  float part[32];
#pragma unroll
  for (int i = 0; i < 32; ++i) {
    const int p = rs_half + 2 * i;
    part[i] = (rs_row < T && p < np) ? rs_src[(int64_t)p * T] : 0.f;
  }
  f32x4 acc[C::FM][C::FN];
  pipe_mainloop<C>(A, B, d, (bf16*)smem, acc);
  {
    float sum = 0.f;
#pragma unroll
    for (int i = 0; i < 32; ++i) sum += part[i];
    if (rs_row < T)
      for (int p = 64 + rs_half; p < np; p += 2) sum += rs_src[(int64_t)p * T];
    sum += __shfl_xor(sum, 1, WAVE);
    if (rs_half == 0) rs_lds[rs_r] = rsqrtf(sum / (float)d + eps);
  }

  // Epilogue through LDS: every wave writes its scaled 64 x 128 tile as bf16 rows (pitch padded
  // by 16 B so the 16 rows written together hit distinct banks), then stores whole 16-byte
  // pieces: 16 lanes cover one 256-byte row, which lies inside one head of Kv or Vv.
  const int lane = threadIdx.x & 63, wave = wave_index();
  const int wm = wave / C::WGN, wn = wave % C::WGN;
  constexpr int EP = kKvEpiPitch;  // bytes per staged row
  unsigned char* ep = smem + wave * (C::WM * EP);
  __syncthreads();  // every wave is done with the pipeline stages
#pragma unroll
  for (int a = 0; a < C::FM; ++a) {
    const int rw = a * 16 + pipe_row(lane);  // row inside the wave tile
    const float rs = rs_lds[wm * C::WM + rw];
#pragma unroll
    for (int b = 0; b < C::FN; ++b) {
      const f32x4& v = acc[a][b];
      const int cw = b * 16 + pipe_col(lane);  // first of this lane's 4 columns in the wave tile
      float y[4] = {v[0] * rs, v[1] * rs, v[2] * rs, v[3] * rs};
      if constexpr (EPI) {
        const int n = n0 + wn * C::WN + cw;
        const bf16* bias = n < kv ? epi.kb : epi.vb;
        if (bias && n < N) {
          float bb[4];
          load4_bf16(bias + (int64_t)l * kv + (n < kv ? n : n - kv), bb);
#pragma unroll
          for (int u = 0; u < 4; ++u) y[u] += bb[u];
        }
      }
      bf16x4 o = {(bf16)y[0], (bf16)y[1], (bf16)y[2], (bf16)y[3]};
      *(u32x2*)(ep + rw * EP + cw * 2) = __builtin_bit_cast(u32x2, o);
    }
  }
  __builtin_amdgcn_s_waitcnt(waitcnt_imm(63, 0));  // this wave's LDS writes landed
  const int64_t head_stride = (int64_t)Nv * hd;
  constexpr int LPR = C::WN / 8;        // lanes per row (8 bf16 each)
  constexpr int RPI = WAVE / LPR;       // rows per store instruction
  const int cpiece = (lane % LPR) * 8;  // first column of this lane's piece
#pragma unroll 4
  for (int r0 = 0; r0 < C::WM; r0 += RPI) {
    const int rw = r0 + lane / LPR;
    const int row = m0 + wm * C::WM + rw;
    const int n = n0 + wn * C::WN + cpiece;
    const bool valid = row < T && n < N;
    u32x4 v = *(const u32x4*)(ep + rw * EP + cpiece * 2);
    if constexpr (EPI) {
      if (epi.kn || epi.rope) {  // uniform: every lane takes the same branch
        const bool is_k = n < kv;
        const int ch = (is_k ? n : n - kv) % hd;  // channel of this lane's first column in its head
        const int half = hd >> 1;
        float x[8];
        unpack8(v, x);
        float sc = 1.f;
        if (epi.kn) {
          // Sum of squares over the head: hd/8 lanes hold one head row (16 for hd 128, 8 for 64).
          float ss = 0.f;
          if (is_k && valid)
#pragma unroll
            for (int e = 0; e < 8; ++e) ss += x[e] * x[e];
          ss += shfl_xor(ss, 1);
          ss += shfl_xor(ss, 2);
          ss += shfl_xor(ss, 4);
          if (hd == 128) ss += shfl_xor(ss, 8);
          sc = rsqrtf(ss / (float)hd + epi.kn_eps);
        }
        if (is_k && valid) {
          if (epi.kn) {
            float w[8];
            unpack8(*(const u32x4*)(epi.kn + (int64_t)l * hd + ch), w);
#pragma unroll
            for (int e = 0; e < 8; ++e) x[e] *= sc * w[e];
          }
          if (epi.rope) {
            const bool first = ch < half;
            const int pc = first ? ch + half : ch - half;  // partner channels of this piece
            float xp[8];
            unpack8(*(const u32x4*)(ep + rw * EP + (cpiece + pc - ch) * 2), xp);
            if (epi.kn) {
              float w[8];
              unpack8(*(const u32x4*)(epi.kn + (int64_t)l * hd + pc), w);
#pragma unroll
              for (int e = 0; e < 8; ++e) xp[e] *= sc * w[e];
            }
            const int j0 = first ? ch : pc;
            const f32x4* cs = (const f32x4*)(epi.rope + ((int64_t)row * half + j0) * 2);
#pragma unroll
            for (int e2 = 0; e2 < 4; ++e2) {
              const f32x4 t = cs[e2];  // (cos, sin) of frequencies j0 + 2 e2 and j0 + 2 e2 + 1
#pragma unroll
              for (int u = 0; u < 2; ++u) {
                const int e = 2 * e2 + u;
                const float c = t[2 * u], sn = t[2 * u + 1];
                x[e] = first ? x[e] * c - xp[e] * sn : x[e] * c + xp[e] * sn;
              }
            }
          }
          v = pack8(x);
        }
      }
    }
    if (!valid) continue;
    const int bb = row / Nv, ii = row - bb * Nv;
    bf16* out = n < kv ? Kv : Vv;
    const int o = n < kv ? n : n - kv;
    const int h = o / hd, c = o - h * hd;
    bf16* dst = out + ((int64_t)l * B_ + bb) * Hkv * head_stride + (int64_t)h * head_stride +
                (int64_t)ii * hd + c;
    __builtin_nontemporal_store(v, (u32x4*)dst);  // streaming: the caches are read by later launches
  }
}

// Backbone epilogue as a pass over stored K/V rows, for the paths whose projection kernel does
// not fuse it (fp32, and bf16 with r not a multiple of 64). One row of hd channels per hd/2
// lanes: lane j holds the rotary pair (j, j + hd/2) of K (and of V for the bias). The row is
// read from the call dtype and rounded once at the end.
template <typename T, int HD>
__global__ __launch_bounds__(256) void k_kv_epi_post(T* __restrict__ Kv, T* __restrict__ Vv,
                                                     int B_, int Nv, int Hkv, int l0, int nl,
                                                     KvEpi<T> epi) {
  constexpr int HALF = HD / 2, RPW = WAVE / HALF;  // rows per wave
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int64_t rows = (int64_t)nl * B_ * Hkv * Nv;
  const int64_t row = ((int64_t)blockIdx.x * 4 + wave) * RPW + lane / HALF;
  const int j = lane % HALF;
  const bool valid = row < rows;
  const int64_t rr = valid ? row : 0;
  const int i = (int)(rr % Nv);
  const int h = (int)((rr / Nv) % Hkv);
  const int b = (int)((rr / ((int64_t)Nv * Hkv)) % B_);
  const int l = l0 + (int)(rr / ((int64_t)Nv * Hkv * B_));
  const int kv = Hkv * HD;
  const int64_t at = ((((int64_t)l * B_ + b) * Hkv + h) * Nv + i) * HD;
  float k1 = 0.f, k2 = 0.f;
  if (valid) {
    k1 = to_f32(Kv[at + j]);
    k2 = to_f32(Kv[at + j + HALF]);
    if (epi.kb) {
      k1 += to_f32(epi.kb[(int64_t)l * kv + h * HD + j]);
      k2 += to_f32(epi.kb[(int64_t)l * kv + h * HD + j + HALF]);
    }
    if (epi.vb) {
      const float v1 = to_f32(Vv[at + j]) + to_f32(epi.vb[(int64_t)l * kv + h * HD + j]);
      const float v2 = to_f32(Vv[at + j + HALF]) + to_f32(epi.vb[(int64_t)l * kv + h * HD + j + HALF]);
      Vv[at + j] = from_f32<T>(v1);
      Vv[at + j + HALF] = from_f32<T>(v2);
    }
  }
  if (epi.kn) {  // uniform
    float ss = k1 * k1 + k2 * k2;
#pragma unroll
    for (int m = 1; m < HALF; m <<= 1) ss += shfl_xor(ss, m);
    const float sc = rsqrtf(ss / (float)HD + epi.kn_eps);
    if (valid) {
      k1 *= sc * to_f32(epi.kn[(int64_t)l * HD + j]);
      k2 *= sc * to_f32(epi.kn[(int64_t)l * HD + j + HALF]);
    }
  }
  if (!valid) return;
  if (epi.rope) {
    const f32x2 cs = *(const f32x2*)(epi.rope + (((int64_t)b * Nv + i) * HALF + j) * 2);
    const float a = k1 * cs[0] - k2 * cs[1];
    k2 = k2 * cs[0] + k1 * cs[1];
    k1 = a;
  }
  if (epi.kb || epi.kn || epi.rope) {
    Kv[at + j] = from_f32<T>(k1);
    Kv[at + j + HALF] = from_f32<T>(k2);
  }
}

// (cos, sin) of the rotary angle for every (token, frequency); fp64 angle and functions.
__global__ __launch_bounds__(256) void k_rope_table(const int32_t* __restrict__ pos, int B_, int Nv,
                                                    int half, int s0, int s1, double log_theta,
                                                    float* __restrict__ table) {
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  const int64_t n = (int64_t)B_ * Nv * half;
  if (idx >= n) return;
  const int j = (int)(idx % half);
  const int64_t t = idx / half;
  const int b = (int)(t / Nv), i = (int)(t - (int64_t)b * Nv);
  const int a = j < s0 ? 0 : (j < s0 + s1 ? 1 : 2);
  const double p = (double)pos[((int64_t)b * 3 + a) * Nv + i];
  const double ang = p * exp(-(double)j / (double)half * log_theta);
  double sn, cs;
  sincos(ang, &sn, &cs);
  *(f32x2*)(table + idx * 2) = f32x2{(float)cs, (float)sn};
}

hipError_t launch_rope_table(const int32_t* pos, int B_, int Nv, int hd, int s0, int s1,
                             float theta, float* table, hipStream_t s) {
  const int half = hd / 2;
  const int64_t n = (int64_t)B_ * Nv * half;
  k_rope_table<<<(unsigned)((n + 255) / 256), 256, 0, s>>>(pos, B_, Nv, half, s0, s1,
                                                          log((double)theta), table);
  return hipGetLastError();
}

template <typename T>
static hipError_t epi_post_launch(void* Kv, void* Vv, int B_, int Nv, int Hkv, int hd, int l0,
                                  int nl, const KvEpiArgs* a, hipStream_t s) {
  const int64_t rows = (int64_t)nl * B_ * Hkv * Nv;
  const int rows_per_block = 4 * (WAVE / (hd / 2));
  const unsigned grid = (unsigned)((rows + rows_per_block - 1) / rows_per_block);
  if (hd == 128)
    k_kv_epi_post<T, 128><<<grid, 256, 0, s>>>((T*)Kv, (T*)Vv, B_, Nv, Hkv, l0, nl, epi_dev<T>(a));
  else
    k_kv_epi_post<T, 64><<<grid, 256, 0, s>>>((T*)Kv, (T*)Vv, B_, Nv, Hkv, l0, nl, epi_dev<T>(a));
  return hipGetLastError();
}

template <typename K>
static void allow_lds(K kernel, int bytes) {
  (void)hipFuncSetAttribute((const void*)kernel, hipFuncAttributeMaxDynamicSharedMemorySize, bytes);
}

// ---------------------------------------------------------------- launchers

// Supertile shapes of the pipelined down and up projections (see supertile_order).
struct TileOrder {
  int sh, sw;
};
static TileOrder down_order() { return TileOrder{8, 8}; }
static TileOrder up_order() { return TileOrder{8, 8}; }

// Layers per block of the tiled up projection. A block reads its tile of E once for all its
// layers and runs them through one pipeline, which saves E reads and block starts; fewer, longer
// blocks balance worse over the CUs. Measured (ms, per step): Qwen2.5-VL video 2.27 with 4
// layers, 2.18 with 8, 2.28-2.40 with 14, 16 or 28; LLaVA-7B 0.31 with 4 or 8, 0.33 with 16.
static int up_layers_per_block(int64_t tiles_per_layer, int nl) {
  (void)tiles_per_layer;
  return std::min(nl, 8);
}

static inline int cdiv(int64_t a, int64_t b) { return (int)((a + b - 1) / b); }

template <typename T>
static hipError_t down_launch(const void* E, const void* Dw, void* Z, int T_, int d, int L, int r,
                              int act, hipStream_t s, const LaunchEvents& ev) {
  typedef typename BuildTiles<T>::Down C;
  dim3 grid(cdiv((int64_t)L * r, C::BN), cdiv(T_, C::BM));
  record(ev.down[0], s);
  if (act == 0)
    k_down_act<C, 0><<<grid, dim3(C::NT), C::LDS_BYTES, s>>>((const T*)E, (const T*)Dw, (T*)Z, T_, d, L, r);
  else
    k_down_act<C, 1><<<grid, dim3(C::NT), C::LDS_BYTES, s>>>((const T*)E, (const T*)Dw, (T*)Z, T_, d, L, r);
  record(ev.down[1], s);
  return hipGetLastError();
}

hipError_t launch_down_act(const void* E, const void* Dw, void* Z, int64_t T_, int d, int L,
                           int r, int act, int dtype, hipStream_t s, const LaunchEvents& ev) {
  if (dtype == 1) {
    // Three tile shapes; each is priced as rounds of its block slots times the outputs a CU
    // computes per round, and the cheapest wins, ties going to the larger tile (fewer operand
    // bytes per MFMA): 256 x 256 (one block per CU), 192 x 128 with eight waves and 128 x 128
    // with four (two blocks per CU each; two 192 x 128 blocks take all 160 KiB of LDS, and forcing
    // one per CU made them 25-35% slower). LLaVA-7B's 2304 x 8192 takes 1.5 rounds of 192 x 128
    // (0.180 -> 0.149 ms against the earlier 96 x 128 blocks, bit-identical), LLaVA-NeXT's 23040 x
    // 8192 15 rounds of 192 x 128 instead of 11.25 of 256 x 256 (1.47 -> 1.31-1.41 ms), and
    // Qwen2.5-VL video's 16384 x 14336 14 whole rounds of 256 x 256.
    static bool once = [] {
      allow_lds(k_down_act_p<KvP, 0>, KvP::LDS_BYTES);
      allow_lds(k_down_act_p<KvP, 1>, KvP::LDS_BYTES);
      allow_lds(k_down_act_p<DownP192, 0>, DownP192::LDS_BYTES);
      allow_lds(k_down_act_p<DownP192, 1>, DownP192::LDS_BYTES);
      return true;
    }();
    (void)once;
    const int64_t N = (int64_t)L * r;
    const int64_t c256 = (int64_t)cdiv(cdiv(N, KvP::BN) * cdiv(T_, KvP::BM), 256) * 256 * 256;
    const int64_t c192 =
        (int64_t)cdiv(cdiv(N, DownP192::BN) * cdiv(T_, DownP192::BM), 512) * 2 * 192 * 128;
    const int64_t c128 = (int64_t)cdiv(cdiv(N, DownP::BN) * cdiv(T_, DownP::BM), 512) * 2 * 128 * 128;
    const bool big = c256 <= c192 && c256 <= c128;
    const bool rows192 = !big && c192 <= c128;
    const TileOrder ord = down_order();
    record(ev.down[0], s);
    if (big) {
      dim3 grid(cdiv(N, KvP::BN), cdiv(T_, KvP::BM));
      if (act == 0)
        k_down_act_p<KvP, 0><<<grid, dim3(KvP::NT), KvP::LDS_BYTES, s>>>((const bf16*)E, (const bf16*)Dw,
                                                                         (bf16*)Z, (int)T_, d, L, r, ord.sh, ord.sw);
      else
        k_down_act_p<KvP, 1><<<grid, dim3(KvP::NT), KvP::LDS_BYTES, s>>>((const bf16*)E, (const bf16*)Dw,
                                                                         (bf16*)Z, (int)T_, d, L, r, ord.sh, ord.sw);
    } else if (rows192) {
      dim3 grid(cdiv(N, DownP192::BN), cdiv(T_, DownP192::BM));
      if (act == 0)
        k_down_act_p<DownP192, 0><<<grid, dim3(DownP192::NT), DownP192::LDS_BYTES, s>>>(
            (const bf16*)E, (const bf16*)Dw, (bf16*)Z, (int)T_, d, L, r, ord.sh, ord.sw);
      else
        k_down_act_p<DownP192, 1><<<grid, dim3(DownP192::NT), DownP192::LDS_BYTES, s>>>(
            (const bf16*)E, (const bf16*)Dw, (bf16*)Z, (int)T_, d, L, r, ord.sh, ord.sw);
    } else {
      dim3 grid(cdiv(N, DownP::BN), cdiv(T_, DownP::BM));
      if (act == 0)
        k_down_act_p<DownP, 0><<<grid, dim3(DownP::NT), DownP::LDS_BYTES, s>>>(
            (const bf16*)E, (const bf16*)Dw, (bf16*)Z, (int)T_, d, L, r, ord.sh, ord.sw);
      else
        k_down_act_p<DownP, 1><<<grid, dim3(DownP::NT), DownP::LDS_BYTES, s>>>(
            (const bf16*)E, (const bf16*)Dw, (bf16*)Z, (int)T_, d, L, r, ord.sh, ord.sw);
    }
    record(ev.down[1], s);
    return hipGetLastError();
  }
  return down_launch<float>(E, Dw, Z, (int)T_, d, L, r, act, s, ev);
}

// Tile order of the K/V projection (see kv_tile). Bytes fetched from beyond the L2s per layer,
// counting an operand tile once per XCD that holds blocks of it: in launch order M * gamma is
// fetched by up to 8 XCDs and the weights by one; with the row tiles dealt out, the reverse.
// Dealing rows out only pays when an XCD's 32 concurrent blocks still span several row tiles
// (at most 8 column tiles): with 32 column tiles they would stream 32 weight tiles at once, and
// the LLaVA-NeXT projection measured 9% slower that way despite the smaller count; the Qwen
// video projection (4 column tiles) measured 1.5% faster.
static int kv_rows_by_xcd(int T_, int d, int N) {
  const int64_t a_bytes = (int64_t)T_ * d * 2, b_bytes = (int64_t)N * d * 2;
  const int64_t n_col = cdiv(N, KvP::BN), n_row = cdiv(T_, KvP::BM);
  if (n_col > 8) return 0;
  const int64_t launch_order = a_bytes * std::min<int64_t>(8, n_col) + b_bytes;
  const int64_t rows_dealt = a_bytes + b_bytes * std::min<int64_t>(8, n_row);
  return rows_dealt < launch_order ? 1 : 0;
}

int kv_partials(int d, int r, int dtype) {
  if (dtype == 1) return r % 64 == 0 ? cdiv(d, UpP::BN) : cdiv(d, BuildTiles<bf16>::Up::BN);
  return cdiv(d, BuildTiles<float>::Up::BN);
}

int kv_partials_max(int d) { return cdiv(d, 64); }

hipError_t launch_kv_only(const void* Mg, const float* ssq, const void* Wk, const void* Wv,
                          void* Kv, void* Vv, int B_, int Nv, int d, int Hkv, int hd, int l0, int nl,
                          int np, float eps, int dtype, hipStream_t s, const LaunchEvents& ev) {
  const int T_ = B_ * Nv;
  if (dtype == 1) {
    static bool once = [] {
      allow_lds(k_kv_proj_p<false>, kKvLdsBytes);
      return true;
    }();
    (void)once;
    dim3 gk(cdiv(2 * Hkv * hd, KvP::BN), cdiv(T_, KvP::BM), nl);
    record(ev.kv[0], s);
    k_kv_proj_p<false><<<gk, dim3(KvP::NT), kKvLdsBytes, s>>>(
        (const bf16*)Mg, ssq, (const bf16*)Wk, (const bf16*)Wv, (bf16*)Kv, (bf16*)Vv, B_, Nv, d,
        Hkv, hd, l0, np, eps, epi_dev<bf16>(nullptr), kv_rows_by_xcd(T_, d, 2 * Hkv * hd));
    record(ev.kv[1], s);
    return hipGetLastError();
  }
  typedef typename BuildTiles<float>::KV CK;
  dim3 gk(cdiv(2 * Hkv * hd, CK::BN), cdiv(T_, CK::BM), nl);
  record(ev.kv[0], s);
  k_kv_proj<CK><<<gk, dim3(CK::NT), CK::LDS_BYTES, s>>>((const float*)Mg, ssq, (const float*)Wk,
                                                         (const float*)Wv, (float*)Kv, (float*)Vv,
                                                         B_, Nv, d, Hkv, hd, l0, np, eps);
  record(ev.kv[1], s);
  return hipGetLastError();
}

static std::atomic<int> g_up_kernel{0};
void set_up_kernel(int mode) { g_up_kernel.store(mode, std::memory_order_relaxed); }

bool up_z_resident(int64_t T, int d, int r, int nl) {
  const int mode = g_up_kernel.load(std::memory_order_relaxed);
  if (mode == 1 || (r != 256 && r != 512)) return false;
  // 32-bit buffer offsets: E, M * gamma and Z_l within 2^31 bytes, U_l below the out-of-range
  // offset of the tile stream.
  if (T * d * 2 >= (int64_t(1) << 31) || T * r * 2 >= (int64_t(1) << 31) ||
      (int64_t)d * r * 2 >= (int64_t(1) << 30))
    return false;
  if (mode == 2) return true;
  // By shape: r = 256 with at least eight rounds of 256 blocks (LLaVA-NeXT: 2.88 -> 2.73 ms).
  // At r = 512 the tiled kernel is faster (Qwen2.5-VL video 2.24 against 2.34 ms), and a few
  // rounds leave too large a tail for blocks that each walk all of d.
  return r == 256 && (int64_t)cdiv(T, upz::BM) * nl >= 8 * 256;
}

static hipError_t kv_launch_bf16(const void* E, const void* Z, const void* Uw, const void* gamma,
                                 const void* Wk, const void* Wv, void* Kv, void* Vv, int B_,
                                 int Nv, int d, int r, int Hkv, int hd, int l0, int nl, float eps,
                                 void* Mg, float* ssq, hipStream_t s, const LaunchEvents& ev,
                                 bool first, bool last, const KvEpiArgs* epi) {
  constexpr int kv_lds = kKvLdsBytes;  // stages (or epilogue staging) + row scales
  static_assert(KvP::NT == 2 * KvP::BM, "two threads per row finish the row scales");
  static bool once = [] {
    allow_lds(k_kv_proj_p<false>, kv_lds);
    allow_lds(k_kv_proj_p<true>, kv_lds);
    allow_lds(k_up_norm_p<UpP>, UpLds<UpP>::BYTES);
    allow_lds(k_up_norm_zr<256>, upz::LDS_BYTES);
    allow_lds(k_up_norm_zr<512>, upz::LDS_BYTES);
    return true;
  }();
  (void)once;
  if (up_kv_fused(d, r, Hkv, hd, 1, epi && epi->any())) {
    // M, its norm and the projection in one kernel (timed as the K/V projection)
    if (first) record(ev.kv[0], s);
    const hipError_t e = launch_up_kv_fused(E, Z, Uw, gamma, Wk, Wv, Kv, Vv, B_, Nv, d, r, Hkv,
                                            hd, l0, nl, eps, s);
    if (last) record(ev.kv[1], s);
    return e;
  }
  const int T_ = B_ * Nv;
  const bool zres = up_z_resident(T_, d, r, nl);
  const int np = zres ? 1 : cdiv(d, UpP::BN);  // sums of squares per row
  if (first) record(ev.up[0], s);
  if (zres) {
    const dim3 gz((unsigned)(cdiv(T_, upz::BM) * nl));
    if (r == 512)
      k_up_norm_zr<512><<<gz, dim3(upz::NW * 64), upz::LDS_BYTES, s>>>(
          (const bf16*)E, (const bf16*)Z, (const bf16*)Uw, (const bf16*)gamma, (bf16*)Mg, ssq, T_,
          d, l0, nl);
    else
      k_up_norm_zr<256><<<gz, dim3(upz::NW * 64), upz::LDS_BYTES, s>>>(
          (const bf16*)E, (const bf16*)Z, (const bf16*)Uw, (const bf16*)gamma, (bf16*)Mg, ssq, T_,
          d, l0, nl);
  } else {
    const int lpb = up_layers_per_block((int64_t)np * cdiv(T_, UpP::BM), nl);
    dim3 gu(np, cdiv(T_, UpP::BM), cdiv(nl, lpb));
    const TileOrder uo = up_order();
    k_up_norm_p<UpP><<<gu, dim3(UpP::NT), UpLds<UpP>::BYTES, s>>>(
        (const bf16*)E, (const bf16*)Z, (const bf16*)Uw, (const bf16*)gamma, (bf16*)Mg, ssq, T_,
        d, r, l0, nl, lpb, uo.sh, uo.sw);
  }
  if (last) record(ev.up[1], s);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  dim3 gk(cdiv(2 * Hkv * hd, KvP::BN), cdiv(T_, KvP::BM), nl);
  if (first) record(ev.kv[0], s);
  if (epi && epi->any())
    k_kv_proj_p<true><<<gk, dim3(KvP::NT), kv_lds, s>>>(
        (const bf16*)Mg, ssq, (const bf16*)Wk, (const bf16*)Wv, (bf16*)Kv, (bf16*)Vv, B_, Nv, d,
        Hkv, hd, l0, np, eps, epi_dev<bf16>(epi), kv_rows_by_xcd(T_, d, 2 * Hkv * hd));
  else
    k_kv_proj_p<false><<<gk, dim3(KvP::NT), kv_lds, s>>>(
        (const bf16*)Mg, ssq, (const bf16*)Wk, (const bf16*)Wv, (bf16*)Kv, (bf16*)Vv, B_, Nv, d,
        Hkv, hd, l0, np, eps, epi_dev<bf16>(nullptr), kv_rows_by_xcd(T_, d, 2 * Hkv * hd));
  if (last) record(ev.kv[1], s);
  return hipGetLastError();
}

template <typename T>
static hipError_t kv_launch(const void* E, const void* Z, const void* Uw, const void* gamma,
                            const void* Wk, const void* Wv, void* Kv, void* Vv, int B_, int Nv,
                            int d, int r, int Hkv, int hd, int l0, int nl, float eps, void* Mg,
                            float* ssq, hipStream_t s, const LaunchEvents& ev, bool first,
                            bool last, const KvEpiArgs* epi) {
  typedef typename BuildTiles<T>::Up CU;
  typedef typename BuildTiles<T>::KV CK;
  const int T_ = B_ * Nv;
  const int np = cdiv(d, CU::BN);
  dim3 gu(np, cdiv(T_, CU::BM), nl);
  if (first) record(ev.up[0], s);
  k_up_norm<CU><<<gu, dim3(CU::NT), CU::LDS_BYTES, s>>>((const T*)E, (const T*)Z, (const T*)Uw, (const T*)gamma, (T*)Mg, ssq, T_, d, r, l0);
  if (last) record(ev.up[1], s);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  dim3 gk(cdiv(2 * Hkv * hd, CK::BN), cdiv(T_, CK::BM), nl);
  if (first) record(ev.kv[0], s);
  k_kv_proj<CK><<<gk, dim3(CK::NT), CK::LDS_BYTES, s>>>((const T*)Mg, ssq, (const T*)Wk, (const T*)Wv, (T*)Kv, (T*)Vv, B_, Nv, d, Hkv, hd, l0, np, eps);
  if (last) record(ev.kv[1], s);
  e = hipGetLastError();
  if (e != hipSuccess || !epi || !epi->any()) return e;
  return epi_post_launch<T>(Kv, Vv, B_, Nv, Hkv, hd, l0, nl, epi, s);
}

hipError_t launch_project_kv(const void* E, const void* Z, const void* Uw, const void* gamma,
                             const void* Wk, const void* Wv, void* Kv, void* Vv, int B_, int Nv,
                             int d, int r, int Hkv, int hd, int l0, int nl, float eps, int dtype,
                             void* Mg, float* ssq, hipStream_t s, const LaunchEvents& ev,
                             bool first, bool last, const KvEpiArgs* epi) {
  if (dtype == 1 && r % 64 == 0)
    return kv_launch_bf16(E, Z, Uw, gamma, Wk, Wv, Kv, Vv, B_, Nv, d, r, Hkv, hd, l0, nl, eps, Mg,
                          ssq, s, ev, first, last, epi);
  if (dtype == 1)
    return kv_launch<bf16>(E, Z, Uw, gamma, Wk, Wv, Kv, Vv, B_, Nv, d, r, Hkv, hd, l0, nl, eps,
                           Mg, ssq, s, ev, first, last, epi);
  return kv_launch<float>(E, Z, Uw, gamma, Wk, Wv, Kv, Vv, B_, Nv, d, r, Hkv, hd, l0, nl, eps,
                          Mg, ssq, s, ev, first, last, epi);
}

}  // namespace dv
