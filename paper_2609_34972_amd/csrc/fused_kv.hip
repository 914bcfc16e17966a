// Fused up-projection, residual, RMSNorm and K/V projection for narrow K/V widths (gfx950).
//
//   Section 3.1 Eq. 4-5:  M_l = E + Z_l U_l            (Z_l = phi(E D_l) from the down projection)
//   Section 3.2 Eq. 7:    [Kv | Vv] = RMSNorm_l(M_l) [Wk_l | Wv_l]^T, stored head-major
//
// When 2 Hkv hd = 1024 (Qwen2.5-VL: 4 K/V heads of 128 channels), the K/V accumulators of 64
// tokens for every output column (64 x 1024 fp32, 256 KiB) fit in half of a CU's register file.
// One block of 4 waves (one per SIMD, each with 256 accumulator registers for its 64 x 256 tile
// and 256 registers for everything else) then owns 64 tokens of one layer and walks d in chunks
// of 64 columns:
//
//   A  M chunk (64 tokens x 64 columns of d) = Z_l rows x a chunk of U_l rows, plus E, in fp32.
//      The 64 rows of Z_l stay in LDS for the whole block; the U_l chunk is staged through LDS.
//      Each wave computes a 32 x 32 quarter of the chunk (fragment reads run two K steps ahead of
//      the MFMAs), adds its row sums of M^2 to two registers and writes bf16(M * gamma) to a
//      64 x 64 LDS tile.
//   B  Every wave multiplies that tile by its 256 columns of [Wk | Wv]. The weight fragments
//      are loaded from memory straight into registers, each refilled with the next chunk's
//      fragment as soon as its MFMAs have been issued; the next U_l chunk streams into LDS
//      meanwhile.
//
// M is produced once per token and never leaves the CU: the two-kernel path writes M * gamma
// (bf16) and fp32 partial sums of squares to HBM and reads them back, 2 x 117 MB per layer at
// the Qwen video shape. The rounding points are those of the two-kernel path (M in fp32, M *
// gamma rounded to bf16 before the projection, the row scale applied to the fp32 product); only
// the order of the row sum of squares differs. The block ends with a staged head-major store of
// whole 16-byte pieces, as in the two-kernel path.
//
// LDS, for rank R: Z rows (64 x R bf16) | U chunk (64 x R) | M * gamma tile (64 x 64) | row sums.
// Rows of Z and U are R * 2 bytes; their 16-byte pieces sit at slot (piece ^ (row % 16)), so the
// 16 rows one fragment read touches fall in 16 distinct bank groups. The M * gamma tile uses the
// 128-byte-row layout of the GEMM pipeline (gemm_pipe.hpp).
#include <atomic>

#include "build_kernels.hpp"
#include "gemm_pipe.hpp"

namespace dv {

namespace {

constexpr int kFRows = 64;    // tokens per block
constexpr int kFCols = 1024;  // K/V columns per block: all of 2 Hkv hd
constexpr int kFChunk = 64;   // columns of d per step

// Block shape for NW waves: each wave owns kFCols / NW K/V columns (all 64 rows) in step B and
// a 32-row x (64 / (NW / 2))-column part of the M chunk in step A.
template <int NW>
struct FusedShape {
  static constexpr int WAVES = NW, THREADS = NW * WAVE;
  static constexpr int WAVE_COLS = kFCols / NW;      // K/V columns per wave
  static constexpr int FN = WAVE_COLS / 16;          // accumulator fragments across them
  static constexpr int W_LOADS = 2 * FN;             // weight fragment loads per chunk
  static constexpr int CGROUPS = NW / 2;             // column groups of the M chunk
  static constexpr int AC = 4 / CGROUPS;             // 16-column fragments per column group
  static constexpr int EPI_PITCH = WAVE_COLS * 2 + 16;  // staged K/V row bytes (padded by 16)
  static constexpr int EPI_BYTES = NW * kFRows * EPI_PITCH;
  static_assert(NW == 4 || NW == 8, "4 or 8 waves");
};

template <int R, int NW>
struct FusedLds {
  static constexpr int ZS = 0;
  static constexpr int US = kFRows * R * 2;
  static constexpr int MS = 2 * kFRows * R * 2;
  static constexpr int MAIN = MS + kFRows * kFChunk * 2;
  static constexpr int EPI = FusedShape<NW>::EPI_BYTES;
  static constexpr int SSX = MAIN > EPI ? MAIN : EPI;  // row sums past the staging area
  static constexpr int BYTES = SSX + FusedShape<NW>::CGROUPS * kFRows * 4;
  static_assert(BYTES <= 160 * 1024, "LDS");
};

__device__ __forceinline__ bf16x8 lds16(const unsigned char* p) {
  return __builtin_bit_cast(bf16x8, *(const u32x4*)p);
}

// 64 rows of R bf16 (row pitch R * 2 bytes in memory too) from `src` + soff into a Z / U tile.
// Rows past the resource's range arrive as zeros. One 1 KiB load covers 64 / (R / 8) rows; lane
// slot s of a row fetches the piece that belongs there, s ^ (row % 16).
template <int R, int NW>
__device__ __forceinline__ void stage_rows(__amdgpu_buffer_rsrc_t src, int soff, unsigned char* dst,
                                           int wave, int lane) {
  constexpr int SPR = R / 8;               // 16-byte slots per row
  constexpr int RPI = WAVE / SPR;          // rows per load
  constexpr int INS = kFRows / RPI / NW;   // loads per wave
  static_assert(SPR >= 16 && WAVE % SPR == 0 && INS >= 1, "rank must be 128, 256 or 512");
  const int slot = lane % SPR, rsub = lane / SPR;
#pragma unroll
  for (int i = 0; i < INS; ++i) {
    const int row0 = (wave * INS + i) * RPI;
    const int row = row0 + rsub;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(src, (lds_void*)(dst + row0 * (2 * R)), 16,
                                             row * (2 * R) + ((slot ^ (row & 15)) << 4), soff, 0,
                                             0);
  }
}

__device__ __forceinline__ u32x4 load16(__amdgpu_buffer_rsrc_t r, int voff, int soff) {
  return __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0));
}
__device__ __forceinline__ u32x2 load8(__amdgpu_buffer_rsrc_t r, int voff, int soff) {
  return __builtin_bit_cast(u32x2, __builtin_amdgcn_raw_buffer_load_b64(r, voff, soff, 0));
}

// The operand pointers are deliberately not __restrict__: the waits before each barrier count
// the loads issued after a given point, so no load may move across the compiler fences around
// the barriers, and loads through a noalias argument may (the fence's memory clobber does not
// reach memory that never escaped).
template <int R, int NW>
__global__ __launch_bounds__(NW * WAVE) __attribute__((amdgpu_waves_per_eu(NW / 4, NW / 4)))
void k_up_kv_fused(const bf16* E, const bf16* Z, const bf16* Uw, const bf16* gamma,
                   const bf16* Wk, const bf16* Wv, bf16* Kv, bf16* Vv, int B_, int Nv, int d,
                   int Hkv, int hd, int l0, float eps, int spread, int step) {
  typedef FusedLds<R, NW> Lo;
  typedef FusedShape<NW> S;
  constexpr int kFWaveCols = S::WAVE_COLS, kFFN = S::FN, kFWLoads = S::W_LOADS;
  constexpr int AC = S::AC, CG = S::CGROUPS;
  constexpr int PD = NW == 4 ? 2 : 1;  // K steps the step-A fragment reads run ahead
  constexpr int KS = R / 32;  // K steps of step A
  extern __shared__ __align__(16) unsigned char smem[];
  unsigned char* zs = smem + Lo::ZS;
  unsigned char* us = smem + Lo::US;
  unsigned char* ms = smem + Lo::MS;
  float* ssx = (float*)(smem + Lo::SSX);
  const int T = B_ * Nv, kv = Hkv * hd;  // kv = kFCols / 2
  const int l = l0 + blockIdx.y;
  const int m0 = blockIdx.x * kFRows;
  const int lane = threadIdx.x & 63, wave = wave_index();
  const int nc = d / kFChunk;

  // Operands as buffer resources: rows past T read as zeros, offsets past the end too.
  const __amdgpu_buffer_rsrc_t zr =
      buffer_rsrc(Z + ((int64_t)l * T + m0) * R, (int64_t)(T - m0) * R * 2);
  const __amdgpu_buffer_rsrc_t ur = buffer_rsrc(Uw + (int64_t)l * d * R, (int64_t)d * R * 2);
  const __amdgpu_buffer_rsrc_t er = buffer_rsrc(E + (int64_t)m0 * d, (int64_t)(T - m0) * d * 2);
  const __amdgpu_buffer_rsrc_t gr = buffer_rsrc(gamma + (int64_t)l * d, (int64_t)d * 2);
  // This wave's output columns: the first half of the waves hold K columns, the rest V columns.
  const bf16* wbase = wave < NW / 2 ? Wk + ((int64_t)l * kv + wave * kFWaveCols) * d
                                    : Wv + ((int64_t)l * kv + (wave - NW / 2) * kFWaveCols) * d;
  const __amdgpu_buffer_rsrc_t wr = buffer_rsrc(wbase, (int64_t)kFWaveCols * d * 2);

  // Step A: rows 32 qr .. +31 and columns 16 AC qc .. of the chunk. Lane l holds token
  // 32 qr + 16 a + l % 16 and columns 16 AC qc + 16 b + 4 (l / 16) .. +3 of fragment (a, b).
  const int qr = wave / CG, qc = wave % CG;
  const int arow = qr * 32 + (lane & 15);
  const int acol = qc * 16 * AC + (lane >> 4) * 4;  // + 16 b
  const int evo = (arow * d + acol) * 2;       // + 16 a rows, + 16 b columns
  // Fragment reads of Z / U rows: every row a lane reads has the same swizzle key l % 16, and
  // K step ks = 4 q + j reads piece 4 ks + l / 16, whose slot is 16 q + ((4 j + l / 16) ^ key).
  // So four per-lane slot offsets plus constant row and q offsets address every read.
  int sj[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) sj[j] = ((4 * j + (lane >> 4)) ^ (lane & 15)) << 4;
  const unsigned char* ub = us + (qc * 16 * AC + (lane & 15)) * (2 * R);  // + 16 b rows
  const unsigned char* zb = zs + arow * (2 * R);                      // + 16 a rows
  // M * gamma tile reads of step B (rows 16 a + l % 16): the slot of piece 4 ks + l / 16 is
  // (4 ks + l / 16) ^ ((l % 16) / 2).
  const unsigned char* mb = ms + (lane & 15) * 128;  // + 2048 a
  const int mk0 = (((lane >> 4)) ^ ((lane & 15) >> 1)) << 4;
  const int mk1 = ((4 + (lane >> 4)) ^ ((lane & 15) >> 1)) << 4;
  // Step B: W fragment b of K step ks of chunk c is row 16 b + l % 16 of the wave's columns,
  // K elements 64 c + 32 ks + 8 (l / 16) .. +7.
  const int wvo = ((lane & 15) * d + (lane >> 4) * 8) * 2;
  // Chunk order. A chunk of the weights is one 128-byte column of rows d * 2 bytes apart, which
  // the L2 interleave maps onto a few of an XCD's channels; blocks that walk d in step would all
  // read those few channels at once. Block x (XCD x % 8 under the dispatcher's round robin)
  // starts at chunk c0 = ((x / 8) % spread) * step and wraps around, so the blocks of an XCD read
  // `spread` different chunks at a time. Step j < nc of the walk is chunk chunk_of(j); j = nc
  // gives -1 (offsets past the end: loads fetch nothing).
  const int c0 = (((int)blockIdx.x >> 3) % spread) * step % nc;
  auto chunk_of = [&](int j) {
    const int c = j + c0;
    return j < nc ? (c < nc ? c : c - nc) : -1;
  };
  auto w_soff = [&](int c, int ks, int b) {
    return c >= 0 ? b * 16 * d * 2 + c * kFChunk * 2 + ks * 64 : kPipeOutOfRange;
  };
  auto load_eg = [&](int c, u32x2 (&e)[2][AC], u32x2 (&g)[AC]) {
    const int soff = c >= 0 ? c * kFChunk * 2 : kPipeOutOfRange;
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
      for (int b = 0; b < AC; ++b) e[a][b] = load8(er, evo + (a * 16 * d + b * 16) * 2, soff);
#pragma unroll
    for (int b = 0; b < AC; ++b) g[b] = load8(gr, (acol + b * 16) * 2, soff);
  };

  f32x4 acc[4][kFFN];
#pragma unroll
  for (int a = 0; a < 4; ++a)
#pragma unroll
    for (int b = 0; b < kFFN; ++b) acc[a][b] = f32x4{};
  float ss[2] = {0.f, 0.f};
  bf16x8 wf[2][kFFN];
  u32x2 e4[2][AC], g4[AC];

  // Prologue: Z rows and U chunk 0 into LDS, E / gamma of chunk 0, all W fragments of chunk 0.
  stage_rows<R, NW>(zr, 0, zs, wave, lane);
  stage_rows<R, NW>(ur, c0 * kFChunk * R * 2, us, wave, lane);
  load_eg(c0, e4, g4);
  asm volatile("" ::: "memory");
#pragma unroll
  for (int ks = 0; ks < 2; ++ks)
#pragma unroll
    for (int b = 0; b < kFFN; ++b)
      wf[ks][b] = __builtin_bit_cast(bf16x8, load16(wr, wvo, w_soff(c0, ks, b)));
  pipe_sync<waitcnt_imm(kFWLoads, 0)>();  // all but the W loads have landed

  for (int j = 0; j < nc; ++j) {
    // ---- A: M chunk part, row sums of squares, bf16(M * gamma) into the LDS tile.
    // Fragment reads run PD K steps ahead of the MFMAs (ring of PD + 1).
    f32x4 am[2][AC];
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
      for (int b = 0; b < AC; ++b) am[a][b] = f32x4{};
    bf16x8 fu[PD + 1][AC], fz[PD + 1][2];
    auto read_step = [&](int ks, int slot) {
      const int off = sj[ks & 3] + (ks >> 2) * 256;
#pragma unroll
      for (int b = 0; b < AC; ++b) fu[slot][b] = lds16(ub + b * 16 * (2 * R) + off);
#pragma unroll
      for (int a = 0; a < 2; ++a) fz[slot][a] = lds16(zb + a * 16 * (2 * R) + off);
    };
#pragma unroll
    for (int ks = 0; ks < PD; ++ks) read_step(ks, ks);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      if (ks + PD < KS) read_step(ks + PD, (ks + PD) % (PD + 1));
      const int s = ks % (PD + 1);
#pragma unroll
      for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int b = 0; b < AC; ++b)
          am[a][b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fu[s][b], fz[s][a], am[a][b], 0, 0, 0);
    }
#pragma unroll
    for (int a = 0; a < 2; ++a) {
      const int row = arow + 16 * a;
#pragma unroll
      for (int b = 0; b < AC; ++b) {
        const bf16x4 e = __builtin_bit_cast(bf16x4, e4[a][b]);
        const bf16x4 g = __builtin_bit_cast(bf16x4, g4[b]);
        bf16x4 o;
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const float m = am[a][b][u] + (float)e[u];
          ss[a] += m * m;
          o[u] = (bf16)(m * (float)g[u]);
        }
        const int k0 = acol + 16 * b;  // column of the chunk
        *(u32x2*)(ms + row * 128 + (((k0 >> 3) ^ ((row >> 1) & 7)) << 4) + (k0 & 7) * 2) =
            __builtin_bit_cast(u32x2, o);
      }
    }
    const int cn = chunk_of(j + 1);
    load_eg(cn, e4, g4);
    // Every wave has written its quarter of the tile and is done reading U chunk c.
    pipe_sync<waitcnt_imm(63, 0)>();
    // Past the last chunk the offset lies beyond U's range: the loads fetch nothing and fill the
    // tile with zeros (not read again). Issuing them anyway keeps the number of loads in flight
    // the same on every iteration, so the compiler's own waits stay tight.
    stage_rows<R, NW>(ur, cn >= 0 ? cn * kFChunk * R * 2 : kPipeOutOfRange, us, wave, lane);
    asm volatile("" ::: "memory");  // the W refills below stay behind the U loads
    // ---- B: K/V accumulators += tile x W chunk c; each W fragment is refilled with chunk c + 1
    // right after its last MFMA.
    bf16x8 mf[2][4];
#pragma unroll
    for (int a = 0; a < 4; ++a) mf[0][a] = lds16(mb + a * 2048 + mk0);
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      if (ks == 0) {
#pragma unroll
        for (int a = 0; a < 4; ++a) mf[1][a] = lds16(mb + a * 2048 + mk1);
      }
#pragma unroll
      for (int b = 0; b < kFFN; ++b) {
#pragma unroll
        for (int a = 0; a < 4; ++a)
          acc[a][b] =
              __builtin_amdgcn_mfma_f32_16x16x32_bf16(wf[ks][b], mf[ks][a], acc[a][b], 0, 0, 0);
        wf[ks][b] = __builtin_bit_cast(bf16x8, load16(wr, wvo, w_soff(cn, ks, b)));
      }
    }
    // U chunk c + 1 (issued before the W refills) has landed; every wave is done with the tile.
    pipe_sync<waitcnt_imm(kFWLoads, 0)>();
  }

  // Row scales: the column groups of each row band meet in LDS (past the staging area).
#pragma unroll
  for (int a = 0; a < 2; ++a) {
    ss[a] += shfl_xor(ss[a], 16);
    ss[a] += shfl_xor(ss[a], 32);
  }
  if (lane < 16) {
    ssx[qc * kFRows + arow] = ss[0];
    ssx[qc * kFRows + arow + 16] = ss[1];
  }
  pipe_sync<waitcnt_imm(0, 0)>();
  float rs[4];
#pragma unroll
  for (int a = 0; a < 4; ++a) {
    const int row = a * 16 + (lane & 15);
    float sum = ssx[row];
#pragma unroll
    for (int g = 1; g < CG; ++g) sum += ssx[g * kFRows + row];
    rs[a] = rsqrtf(sum / (float)d + eps);
  }

  // Staged head-major store: each wave writes its scaled 64 x 256 tile as bf16 rows, then stores
  // whole 16-byte pieces, 32 lanes per 512-byte row (two heads of 128 or four of 64).
  constexpr int kFEpiPitch = S::EPI_PITCH;
  unsigned char* ep = smem + wave * (kFRows * kFEpiPitch);
#pragma unroll
  for (int a = 0; a < 4; ++a) {
    const int rw = a * 16 + (lane & 15);
#pragma unroll
    for (int b = 0; b < kFFN; ++b) {
      const f32x4& v = acc[a][b];
      const int cw = b * 16 + (lane >> 4) * 4;
      bf16x4 o = {(bf16)(v[0] * rs[a]), (bf16)(v[1] * rs[a]), (bf16)(v[2] * rs[a]),
                  (bf16)(v[3] * rs[a])};
      *(u32x2*)(ep + rw * kFEpiPitch + cw * 2) = __builtin_bit_cast(u32x2, o);
    }
  }
  __builtin_amdgcn_s_waitcnt(waitcnt_imm(63, 0));  // this wave's LDS writes landed
  const int64_t head_stride = (int64_t)Nv * hd;
  constexpr int LPR = kFWaveCols / 8;  // lanes per row
  constexpr int RPI = WAVE / LPR;      // rows per store
  const int cpiece = (lane % LPR) * 8;
  const int n = wave * kFWaveCols + cpiece;
  bf16* out = n < kv ? Kv : Vv;
  const int o = n < kv ? n : n - kv;
  const int h = o / hd, ch = o - h * hd;
#pragma unroll 4
  for (int r0 = 0; r0 < kFRows; r0 += RPI) {
    const int rw = r0 + lane / LPR;
    const int row = m0 + rw;
    if (row >= T) continue;
    const u32x4 v = *(const u32x4*)(ep + rw * kFEpiPitch + cpiece * 2);
    const int bb = row / Nv, ii = row - bb * Nv;
    bf16* dst = out + (((int64_t)l * B_ + bb) * Hkv + h) * head_stride + (int64_t)ii * hd + ch;
    __builtin_nontemporal_store(v, (u32x4*)dst);
  }
}

struct FusedOrder {
  int spread, step;
};
static FusedOrder fused_order() { return FusedOrder{16, 1}; }

template <int R, int NW>
hipError_t fused_launch(const void* E, const void* Z, const void* Uw, const void* gamma,
                        const void* Wk, const void* Wv, void* Kv, void* Vv, int B_, int Nv, int d,
                        int Hkv, int hd, int l0, int nl, float eps, hipStream_t s) {
  const FusedOrder ord = fused_order();
  static bool once = [] {
    (void)hipFuncSetAttribute((const void*)k_up_kv_fused<R, NW>,
                              hipFuncAttributeMaxDynamicSharedMemorySize, FusedLds<R, NW>::BYTES);
    return true;
  }();
  (void)once;
  const int64_t T = (int64_t)B_ * Nv;
  dim3 grid((unsigned)((T + kFRows - 1) / kFRows), (unsigned)nl);
  k_up_kv_fused<R, NW><<<grid, dim3(NW * WAVE), FusedLds<R, NW>::BYTES, s>>>(
      (const bf16*)E, (const bf16*)Z, (const bf16*)Uw, (const bf16*)gamma, (const bf16*)Wk,
      (const bf16*)Wv, (bf16*)Kv, (bf16*)Vv, B_, Nv, d, Hkv, hd, l0, eps, ord.spread, ord.step);
  return hipGetLastError();
}

#ifndef DV_FUSED_WAVES
#define DV_FUSED_WAVES 8
#endif
constexpr int kFusedWaves = DV_FUSED_WAVES;

std::atomic<int> g_fused_enabled{0};

}  // namespace

void set_up_kv_fused(bool on) { g_fused_enabled.store(on ? 1 : 0, std::memory_order_relaxed); }

bool up_kv_fused_eligible(int d, int r, int Hkv, int hd, int dtype) {
  return dtype == 1 && (int64_t)2 * Hkv * hd == kFCols && (hd == 64 || hd == 128) &&
         (r == 128 || r == 256 || r == 512) && d % kFChunk == 0 && d > 0;
}

bool up_kv_fused(int d, int r, int Hkv, int hd, int dtype, bool epilogue) {
  return g_fused_enabled.load(std::memory_order_relaxed) != 0 && !epilogue &&
         up_kv_fused_eligible(d, r, Hkv, hd, dtype);
}

hipError_t launch_up_kv_fused(const void* E, const void* Z, const void* Uw, const void* gamma,
                              const void* Wk, const void* Wv, void* Kv, void* Vv, int B_, int Nv,
                              int d, int r, int Hkv, int hd, int l0, int nl, float eps,
                              hipStream_t s) {
  switch (r) {
    case 128:
      return fused_launch<128, kFusedWaves>(E, Z, Uw, gamma, Wk, Wv, Kv, Vv, B_, Nv, d, Hkv, hd, l0, nl, eps, s);
    case 256:
      return fused_launch<256, kFusedWaves>(E, Z, Uw, gamma, Wk, Wv, Kv, Vv, B_, Nv, d, Hkv, hd, l0, nl, eps, s);
    case 512:
      return fused_launch<512, kFusedWaves>(E, Z, Uw, gamma, Wk, Wv, Kv, Vv, B_, Nv, d, Hkv, hd, l0, nl, eps, s);
    default:
      return hipErrorInvalidValue;
  }
}

}  // namespace dv
