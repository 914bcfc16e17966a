// Block-tiled "NT" GEMM main loop for gfx950:  C[m][n] = sum_k A[m][k] * B[n][k].
//
// Both operands are K-contiguous (weights are stored out x in), so every lane
// reads its MFMA fragment as one 16-byte (bf16) or two 16-byte (fp32) LDS
// loads with no transposition. Tiles are staged global -> registers -> LDS
// with two LDS buffers, so the loads of tile k+1 are in flight while the MFMAs
// of tile k run, and only one barrier per K tile is needed.
#pragma once

#include "dv_device.hpp"

namespace dv {

template <typename T, int BM_, int BN_, int WGM_, int WGN_>
struct TileCfg {
  typedef T elem;
  static constexpr int BM = BM_, BN = BN_, WGM = WGM_, WGN = WGN_;
  static constexpr int NT = WAVE * WGM * WGN;
  static constexpr int EPC = 16 / (int)sizeof(T);  // elements per 16-byte chunk
  static constexpr int BK = 8 * EPC;               // 128-byte LDS rows (8 chunks)
  static constexpr int WM = BM / WGM, WN = BN / WGN;
  static constexpr int FM = WM / 32, FN = WN / 32;
  static constexpr int A_IT = BM * 8 / NT, B_IT = BN * 8 / NT;
  static constexpr int STAGE = (BM + BN) * BK;  // elements per LDS stage
  static constexpr int LDS_BYTES = 2 * STAGE * (int)sizeof(T);
  static_assert(WM % 32 == 0 && WN % 32 == 0, "wave tile must be a multiple of 32x32");
  static_assert((BM * 8) % NT == 0 && (BN * 8) % NT == 0, "tile chunks must divide threads");
};

// Eight K-consecutive elements of row `row` starting at element `kel` (a
// multiple of 8) of a swizzled LDS tile with 128-byte rows.
__device__ __forceinline__ bf16x8 lds_frag8(const bf16* s, int row, int kel) {
  const int c = kel >> 3;
  u32x4 v = *(const u32x4*)(s + row * 64 + swz(row, c) * 8);
  return __builtin_bit_cast(bf16x8, v);
}
__device__ __forceinline__ f32x8 lds_frag8(const float* s, int row, int kel) {
  const int c = kel >> 2;
  u32x4 v0 = *(const u32x4*)(s + row * 32 + swz(row, c) * 4);
  u32x4 v1 = *(const u32x4*)(s + row * 32 + swz(row, c + 1) * 4);
  f32x4 a = __builtin_bit_cast(f32x4, v0), b = __builtin_bit_cast(f32x4, v1);
  return f32x8{a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
}

// Row pointer of B: rows [0, nsplit) come from B0, rows [nsplit, N) from B1
// (lets the K and V projections share one N range without a concatenated copy).
template <typename T>
struct BRows {
  const T* B0;
  const T* B1;
  int64_t ldb;
  int nsplit;
  __device__ __forceinline__ const T* row(int n) const {
    return n < nsplit ? B0 + (int64_t)n * ldb : B1 + (int64_t)(n - nsplit) * ldb;
  }
};

template <class C>
__device__ __forceinline__ void gemm_nt_mainloop(const typename C::elem* __restrict__ A,
                                                 int64_t lda, int M, BRows<typename C::elem> B,
                                                 int N, int K, int m0, int n0,
                                                 typename C::elem* lds,
                                                 f32x16 (&acc)[C::FM][C::FN]) {
  typedef typename C::elem T;
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = wave / C::WGN, wn = wave % C::WGN;
  u32x4 ra[C::A_IT], rb[C::B_IT];

#pragma unroll
  for (int a = 0; a < C::FM; ++a)
#pragma unroll
    for (int b = 0; b < C::FN; ++b) acc[a][b] = f32x16{};

  auto gload = [&](int k0) {
#pragma unroll
    for (int i = 0; i < C::A_IT; ++i) {
      const int idx = tid + i * C::NT, row = idx >> 3, ch = idx & 7;
      const int gm = m0 + row, kk = k0 + ch * C::EPC;
      ra[i] = (gm < M && kk < K) ? *(const u32x4*)(A + (int64_t)gm * lda + kk) : u32x4{0, 0, 0, 0};
    }
#pragma unroll
    for (int i = 0; i < C::B_IT; ++i) {
      const int idx = tid + i * C::NT, row = idx >> 3, ch = idx & 7;
      const int gn = n0 + row, kk = k0 + ch * C::EPC;
      rb[i] = (gn < N && kk < K) ? *(const u32x4*)(B.row(gn) + kk) : u32x4{0, 0, 0, 0};
    }
  };
  auto sstore = [&](int buf) {
    T* sa = lds + buf * C::STAGE;
    T* sb = sa + C::BM * C::BK;
#pragma unroll
    for (int i = 0; i < C::A_IT; ++i) {
      const int idx = tid + i * C::NT, row = idx >> 3, ch = idx & 7;
      *(u32x4*)(sa + row * C::BK + swz(row, ch) * C::EPC) = ra[i];
    }
#pragma unroll
    for (int i = 0; i < C::B_IT; ++i) {
      const int idx = tid + i * C::NT, row = idx >> 3, ch = idx & 7;
      *(u32x4*)(sb + row * C::BK + swz(row, ch) * C::EPC) = rb[i];
    }
  };

  const int nk = (K + C::BK - 1) / C::BK;
  gload(0);
  sstore(0);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    if (kt + 1 < nk) gload((kt + 1) * C::BK);
    const T* sa = lds + (kt & 1) * C::STAGE;
    const T* sb = sa + C::BM * C::BK;
#pragma unroll
    for (int ks = 0; ks < C::BK / 16; ++ks) {
      const int kel = ks * 16 + (lane >> 5) * 8;
      typename Frag8<T>::type fa[C::FM], fb[C::FN];
#pragma unroll
      for (int a = 0; a < C::FM; ++a) fa[a] = lds_frag8(sa, wm * C::WM + a * 32 + (lane & 31), kel);
#pragma unroll
      for (int b = 0; b < C::FN; ++b) fb[b] = lds_frag8(sb, wn * C::WN + b * 32 + (lane & 31), kel);
#pragma unroll
      for (int a = 0; a < C::FM; ++a)
#pragma unroll
        for (int b = 0; b < C::FN; ++b) mfma_k16(acc[a][b], fa[a], fb[b]);
    }
    if (kt + 1 < nk) sstore((kt + 1) & 1);
    __syncthreads();
  }
}

}  // namespace dv
