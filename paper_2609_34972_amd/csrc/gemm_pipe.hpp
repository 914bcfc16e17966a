// Software-pipelined bf16 "NT" GEMM main loop for gfx950:  C[m][n] = sum_k A[m][k] * B[n][k].
//
// * Operand tiles go straight from HBM into LDS with buffer_load ... lds (no staging registers).
//   The buffer resources carry the valid byte range, so rows past the end read as zeros instead
//   of faulting.
// * Two 64-deep LDS stages: the loads of tile k+2 are issued as soon as every wave has finished
//   reading tile k, and the next tile's first fragments are read before the last MFMA group of
//   the current tile, so one barrier per K tile carries no exposed LDS latency. Both halves of a
//   tile interleave their memory instructions with MFMAs: before the barrier the second K step's
//   fragment reads, after it the refill loads and the next tile's first fragment reads.
// * Out-of-range buffer loads fetch nothing and write zeros, also into LDS (measured on gfx950,
//   whether the excess offset sits in the vector or the scalar offset).
// * 128-byte LDS rows with an XOR swizzle of the 16-byte chunks keyed on (row / 2) mod 8: the
//   16 rows read together by a fragment load land in 16 distinct bank groups. Lanes of a load
//   instruction pick the global chunk that belongs at their LDS slot, so the swizzle costs
//   nothing at load time.
// * 16x16x32 MFMAs. With random bf16 operands the chip's clock (and so the MFMA rate) falls
//   under load, and it falls less for this shape than for 32x32x16: a register-resident MFMA
//   loop sustains about 1.9 PFLOP/s against 1.72 for 32x32x16 (both about 2.46 with constant
//   operands). Every fragment still is one 16-byte LDS read per lane.
// * The MFMA operands are swapped (acc = B-fragment x A-fragment), which leaves the transpose
//   of the 16x16 tile in the accumulators: lane l holds row m = l % 16 of its fragment and one
//   run of four consecutive columns starting at 4 * (l / 16). Epilogues therefore see one
//   output row per lane and fragment (per-row scales are per lane) and store 8-byte runs along
//   the row.
#pragma once

#include "dv_device.hpp"

namespace dv {

typedef __attribute__((address_space(3))) void lds_void;

// s_waitcnt immediate (gfx9 encoding): at most `vm` vector-memory and `lgkm` LDS/scalar ops
// outstanding, export count not waited on.
constexpr int waitcnt_imm(int vm, int lgkm) {
  return (vm & 0xF) | ((vm >> 4) << 14) | (0x7 << 4) | ((lgkm & 0xF) << 8);
}

constexpr int kRawBufferFlags = 0x00020000;  // dword 3 of a raw (unformatted) buffer resource
// A load offset past every operand buffer's range (they are at most 2^31 - 1 bytes and the
// in-tile offsets stay far below 2^30): such a load fetches nothing and returns zeros.
constexpr int kPipeOutOfRange = 0x40000000;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t buffer_rsrc(const void* base, int64_t bytes) {
  const int nr = bytes > 0x7fffffff ? 0x7fffffff : (bytes < 0 ? 0 : (int)bytes);
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, nr, kRawBufferFlags);
}

// One GEMM operand as row ranges of up to two buffers: rows [0, nsplit) come from r0, rows
// [nsplit, ...) from r1 (row nsplit is r1's first row). Row pitch in bytes.
struct BufOperand {
  __amdgpu_buffer_rsrc_t r0, r1;
  int nsplit;
  int ld_bytes;
};

__device__ __forceinline__ int wave_index() {
  return __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
}

template <int BM_, int BN_, int WGM_, int WGN_>
struct PipeCfg {
  static constexpr int BM = BM_, BN = BN_, WGM = WGM_, WGN = WGN_;
  static constexpr int NWAVES = WGM * WGN, NT = WAVE * NWAVES;
  static constexpr int BK = 64;
  static constexpr int WM = BM / WGM, WN = BN / WGN;
  static constexpr int FM = WM / 16, FN = WN / 16;  // 16x16 accumulator fragments per wave
  static constexpr int A_INS = BM / 8 / NWAVES;  // 8-row (1 KiB) load instructions per wave
  static constexpr int B_INS = BN / 8 / NWAVES;
  static constexpr int INS = A_INS + B_INS;
  static constexpr int STAGE = (BM + BN) * BK;   // bf16 elements per stage
  static constexpr int LDS_BYTES = 2 * STAGE * 2;
  static_assert(WM % 16 == 0 && WN % 16 == 0 && A_INS >= 1 && B_INS >= 1, "bad tile");
};

// Lane byte offset inside an 8-row load block: LDS slot (row r = lane / 8, chunk pc = lane % 8)
// holds logical chunk pc ^ key(row), key(row) = (row / 2) % 8 = (r / 2) | 4 * (block % 2).
__device__ __forceinline__ int pipe_lane_offset(int ld_bytes, int odd_block) {
  const int lane = threadIdx.x & 63, r = lane >> 3, pc = lane & 7;
  const int key = (r >> 1) | (odd_block << 2);
  return r * ld_bytes + ((pc ^ key) << 4);
}

// What a wave's refill loads need besides the K offset, fixed for a whole GEMM: the buffer of
// each B load (the B tile may straddle the two row ranges) and the byte offset of each load's
// 8-row block. Worked out once, so a refill costs one scalar add per load.
struct PipeRsrc {  // (an array of the bare resource type does not compile for the host pass)
  __amdgpu_buffer_rsrc_t r;
};
template <class C>
struct PipeLoads {
  __amdgpu_buffer_rsrc_t ra;
  PipeRsrc rb[C::B_INS];
  int sa[C::A_INS], sb[C::B_INS];
};

template <class C>
__device__ __forceinline__ PipeLoads<C> pipe_loads(const BufOperand& A, const BufOperand& B) {
  PipeLoads<C> p;
  const int wave = wave_index();
  p.ra = A.r0;
#pragma unroll
  for (int i = 0; i < C::A_INS; ++i) p.sa[i] = (wave * C::A_INS + i) * 8 * A.ld_bytes;
#pragma unroll
  for (int i = 0; i < C::B_INS; ++i) {
    const int row = (wave * C::B_INS + i) * 8;
    const bool first = row < B.nsplit;
    p.rb[i].r = first ? B.r0 : B.r1;
    p.sb[i] = (first ? row : row - B.nsplit) * B.ld_bytes;
  }
  return p;
}

// Each wave issues A_INS + B_INS 1 KiB loads (8 rows x 128 bytes) of one 64-deep K tile. A
// load's 8-row block parity selects the swizzle key half; with an even count per wave it is that
// of the load's index, with an odd count it also depends on the wave.
template <int INS>
__device__ __forceinline__ bool pipe_odd_block(int wave, int i) {
  return INS % 2 == 0 ? (i & 1) != 0 : ((wave * INS + i) & 1) != 0;
}

template <class C>
__device__ __forceinline__ void pipe_issue(const PipeLoads<C>& p, int kbytes, bf16* stage, int va0,
                                           int va1, int vb0, int vb1) {
  const int wave = wave_index();
#pragma unroll
  for (int i = 0; i < C::A_INS; ++i) {
    const int blk = wave * C::A_INS + i;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(p.ra, (lds_void*)(stage + blk * 512), 16,
                                             pipe_odd_block<C::A_INS>(wave, i) ? va1 : va0,
                                             p.sa[i] + kbytes, 0, 0);
  }
  bf16* sb = stage + C::BM * C::BK;
#pragma unroll
  for (int i = 0; i < C::B_INS; ++i) {
    const int blk = wave * C::B_INS + i;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(p.rb[i].r, (lds_void*)(sb + blk * 512), 16,
                                             pipe_odd_block<C::B_INS>(wave, i) ? vb1 : vb0,
                                             p.sb[i] + kbytes, 0, 0);
  }
}

__device__ __forceinline__ bf16x8 pipe_frag(const bf16* s, int row, int chunk) {
  const int pc = chunk ^ ((row >> 1) & 7);
  return __builtin_bit_cast(bf16x8, *(const u32x4*)(s + row * 64 + pc * 8));
}

// Fragments of one 32-deep K step ks (0 or 1) of a 64-deep stage: lane l reads row l % 16 of
// each 16-row fragment, K elements 8 * (l / 16) .. +7 of the step.
template <class C>
__device__ __forceinline__ void pipe_frags(const bf16* s, int ks, bf16x8 (&fa)[C::FM],
                                           bf16x8 (&fb)[C::FN]) {
  const int lane = threadIdx.x & 63, wave = wave_index();
  const int wm = wave / C::WGN, wn = wave % C::WGN;
  const int chunk = ks * 4 + (lane >> 4);
  const bf16* sb = s + C::BM * C::BK;
#pragma unroll
  for (int a = 0; a < C::FM; ++a) fa[a] = pipe_frag(s, wm * C::WM + a * 16 + (lane & 15), chunk);
#pragma unroll
  for (int b = 0; b < C::FN; ++b) fb[b] = pipe_frag(sb, wn * C::WN + b * 16 + (lane & 15), chunk);
}

template <class C>
__device__ __forceinline__ void pipe_mfmas(f32x4 (&acc)[C::FM][C::FN], const bf16x8 (&fa)[C::FM],
                                           const bf16x8 (&fb)[C::FN]) {
#pragma unroll
  for (int a = 0; a < C::FM; ++a)
#pragma unroll
    for (int b = 0; b < C::FN; ++b)  // transposed tile
      acc[a][b] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(fb[b], fa[a], acc[a][b], 0, 0, 0);
}

template <int IMM>
__device__ __forceinline__ void pipe_sync() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt(IMM);
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Accumulator item u (0..3) of fragment (a, b) of a wave holds row a*16 + pipe_row(lane) and
// column b*16 + pipe_col(lane) + u of the wave tile.
__device__ __forceinline__ int pipe_row(int lane) { return lane & 15; }
__device__ __forceinline__ int pipe_col(int lane) { return (lane >> 4) * 4; }

// Issue order of the first K step: two MFMAs, then each of the second step's fragment reads
// followed by one MFMA, then the rest (the reads, which the tile barrier waits for, go out early;
// two MFMAs per read, or reads from the first MFMA on, measured equal or slower).
template <class C>
__device__ __forceinline__ void pipe_step0_pattern() {
  static_assert(C::FM * C::FN >= 2 + C::FM + C::FN, "a K step needs an MFMA per fragment read");
  __builtin_amdgcn_sched_group_barrier(0x008, 2, 0);
#pragma unroll
  for (int i = 0; i < C::FM + C::FN; ++i) {
    __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
  }
  __builtin_amdgcn_sched_group_barrier(0x008, C::FM * C::FN - 2 - (C::FM + C::FN), 0);
}

// Issue order of the second K step: the refill loads first, each followed by kPer MFMAs (loads
// spread out went slightly faster than one per MFMA; fragment reads first, slower), then each of
// the next tile's fragment reads followed by one MFMA, then the rest of the MFMAs.
// Tiles with fewer MFMAs per K step than loads plus reads (e.g. 96 x 128) leave the order to the
// compiler.
template <class C>
__device__ __forceinline__ void pipe_step1_pattern() {
  constexpr int kPer = (C::FM * C::FN - (C::FM + C::FN)) / C::INS;
  if constexpr (kPer >= 1) {
#pragma unroll
    for (int i = 0; i < C::INS; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x020, 1, 1);
      __builtin_amdgcn_sched_group_barrier(0x008, kPer, 1);
    }
#pragma unroll
    for (int i = 0; i < C::FM + C::FN; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 1);
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 1);
    }
    __builtin_amdgcn_sched_group_barrier(0x008,
                                         C::FM * C::FN - kPer * C::INS - (C::FM + C::FN), 1);
  }
}

// A: block-tile rows start at A's first row; B likewise. K must be a multiple of 64.
template <class C>
__device__ __forceinline__ void pipe_mainloop(const BufOperand& A, const BufOperand& B, int K,
                                              bf16* lds, f32x4 (&acc)[C::FM][C::FN]) {
#pragma unroll
  for (int a = 0; a < C::FM; ++a)
#pragma unroll
    for (int b = 0; b < C::FN; ++b) acc[a][b] = f32x4{};
  const int va0 = pipe_lane_offset(A.ld_bytes, 0), va1 = pipe_lane_offset(A.ld_bytes, 1);
  const int vb0 = pipe_lane_offset(B.ld_bytes, 0), vb1 = pipe_lane_offset(B.ld_bytes, 1);
  const int nk = K / C::BK;
  const PipeLoads<C> pl = pipe_loads<C>(A, B);
  pipe_issue<C>(pl, 0, lds, va0, va1, vb0, vb1);
  if (nk > 1) {
    pipe_issue<C>(pl, C::BK * 2, lds + C::STAGE, va0, va1, vb0, vb1);
    pipe_sync<waitcnt_imm(C::INS, 0)>();  // tile 0 landed, tile 1 stays in flight
  } else {
    pipe_sync<waitcnt_imm(0, 0)>();
  }
  bf16x8 fa[2][C::FM], fb[2][C::FN];
  pipe_frags<C>(lds, 0, fa[0], fb[0]);
  for (int kt = 0; kt < nk; ++kt) {
    bf16* s = lds + (kt & 1) * C::STAGE;
    // K step 0: the step-1 fragments are read between its MFMAs (pipe_step0_pattern), so the
    // reads overlap the matrix pipe.
    pipe_frags<C>(s, 1, fa[1], fb[1]);
    pipe_mfmas<C>(acc, fa[0], fb[0]);
    pipe_step0_pattern<C>();
    // Keep this step's MFMAs ahead of the barrier (the compiler would otherwise sink them below
    // it, next to their next use), so they cover the fragment reads the barrier waits for.
#pragma unroll
    for (int a = 0; a < C::FM; ++a)
#pragma unroll
      for (int b = 0; b < C::FN; ++b) asm volatile("" : "+v"(acc[a][b]));
    // K step 1: every wave holds its last fragments of stage s and tile kt+1 has landed:
    // refill s with tile kt+2 and fetch tile kt+1's first fragments before this step's MFMAs.
    pipe_sync<waitcnt_imm(0, 0)>();
    // Neither the refill nor the next fragment reads is conditional, so both interleave with
    // this step's MFMAs: past the last tile the refill offset lies beyond the buffers' range
    // (nothing is fetched; the stage, which is not read again, fills with zeros) and the
    // fragments read from a stale stage go unused.
    const int kb2 = kt + 2 < nk ? (kt + 2) * C::BK * 2 : kPipeOutOfRange;
    pipe_issue<C>(pl, kb2, s, va0, va1, vb0, vb1);
    pipe_frags<C>(lds + ((kt + 1) & 1) * C::STAGE, 0, fa[0], fb[0]);
    pipe_mfmas<C>(acc, fa[1], fb[1]);
    pipe_step1_pattern<C>();
    __builtin_amdgcn_sched_barrier(0);  // keeps the two K steps' patterns in separate regions
  }
  // The last tile's zero-filling refill and fragment reads come after the last barrier: every
  // wave's must be complete before any wave goes on to reuse the stages (epilogues may write
  // them without a barrier of their own).
  pipe_sync<waitcnt_imm(0, 0)>();
}

// Refill loads of one K tile of a run's operands. The per-load row offsets (and, for B, the
// buffer of each load) are the same for every run, so they are worked out once per stream.
template <class C>
__device__ __forceinline__ void pipe_issue_rsrc(const PipeLoads<C>& p, const BufOperand& A,
                                                const BufOperand& B, int kbytes, bf16* stage,
                                                int va0, int va1, int vb0, int vb1) {
  const int wave = wave_index();
#pragma unroll
  for (int i = 0; i < C::A_INS; ++i) {
    const int blk = wave * C::A_INS + i;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(A.r0, (lds_void*)(stage + blk * 512), 16,
                                             (blk & 1) ? va1 : va0, p.sa[i] + kbytes, 0, 0);
  }
  bf16* sb = stage + C::BM * C::BK;
#pragma unroll
  for (int i = 0; i < C::B_INS; ++i) {
    const int blk = wave * C::B_INS + i;
    const bool first = blk * 8 < B.nsplit;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(first ? B.r0 : B.r1, (lds_void*)(sb + blk * 512), 16,
                                             (blk & 1) ? vb1 : vb0, p.sb[i] + kbytes, 0, 0);
  }
}

// Several GEMMs of the same K through one pipeline (e.g. one output tile of consecutive layers).
// Tile t of the stream is K tile t % nk of run t / nk, nk = K / 64. operands(run, A, B) fills a
// run's operands (every run has the same row pitches and the same B split row); epilogue(run,
// acc) consumes a finished run while the loads of the next run's first two tiles are in flight,
// so the pipeline does not drain between runs. The epilogue may use LDS past the two stages
// (C::LDS_BYTES) but not the stages themselves, since a landed tile may sit there.
// The refill side keeps the run and K tile of the next tile to load and the operands of that run,
// which it rebuilds only when the run changes: a tile's refill then costs a few scalar adds (a
// division and the operand addresses at every tile put ~55 dependent scalar instructions ahead
// of each tile's first MFMA).
template <class C, class Operands, class Epilogue>
__device__ __forceinline__ void pipe_runs(int nruns, int K, bf16* lds, Operands operands,
                                          Epilogue epilogue) {
  f32x4 acc[C::FM][C::FN];
#pragma unroll
  for (int a = 0; a < C::FM; ++a)
#pragma unroll
    for (int b = 0; b < C::FN; ++b) acc[a][b] = f32x4{};
  const int nk = K / C::BK, nt = nruns * nk;
  BufOperand An, Bn;  // operands of the run of the next tile to load
  operands(0, An, Bn);
  const int va0 = pipe_lane_offset(An.ld_bytes, 0), va1 = pipe_lane_offset(An.ld_bytes, 1);
  const int vb0 = pipe_lane_offset(Bn.ld_bytes, 0), vb1 = pipe_lane_offset(Bn.ld_bytes, 1);
  const PipeLoads<C> pl = pipe_loads<C>(An, Bn);
  int rn = 0, kn = 0;  // run and K tile of the next tile to load
  // Issues the next tile (past the stream's end: out-of-range loads of the last run, which fetch
  // nothing and fill the stage with zeros) and steps to the one after it.
  auto refill = [&](bf16* stage) {
    const int kbytes = rn < nruns ? kn * C::BK * 2 : kPipeOutOfRange;
    pipe_issue_rsrc<C>(pl, An, Bn, kbytes, stage, va0, va1, vb0, vb1);
    if (++kn == nk) {
      kn = 0;
      if (++rn < nruns) operands(rn, An, Bn);
    }
  };

  refill(lds);
  if (nt > 1) {
    refill(lds + C::STAGE);
    pipe_sync<waitcnt_imm(C::INS, 0)>();
  } else {
    pipe_sync<waitcnt_imm(0, 0)>();
  }
  bf16x8 fa[2][C::FM], fb[2][C::FN];
  pipe_frags<C>(lds, 0, fa[0], fb[0]);
  int kk = 0, run = 0;  // K tile of t within its run, and its run
  for (int t = 0; t < nt; ++t) {
    bf16* s = lds + (t & 1) * C::STAGE;
    pipe_frags<C>(s, 1, fa[1], fb[1]);
    pipe_mfmas<C>(acc, fa[0], fb[0]);
    pipe_step0_pattern<C>();
#pragma unroll
    for (int a = 0; a < C::FM; ++a)
#pragma unroll
      for (int b = 0; b < C::FN; ++b) asm volatile("" : "+v"(acc[a][b]));
    pipe_sync<waitcnt_imm(0, 0)>();
    refill(s);
    pipe_frags<C>(lds + ((t + 1) & 1) * C::STAGE, 0, fa[0], fb[0]);
    pipe_mfmas<C>(acc, fa[1], fb[1]);
    pipe_step1_pattern<C>();
    __builtin_amdgcn_sched_barrier(0);
    if (++kk == nk) {
      epilogue(run, acc);
#pragma unroll
      for (int a = 0; a < C::FM; ++a)
#pragma unroll
        for (int b = 0; b < C::FN; ++b) acc[a][b] = f32x4{};
      kk = 0;
      ++run;
    }
  }
  pipe_sync<waitcnt_imm(0, 0)>();  // as at the end of pipe_mainloop
}

}  // namespace dv
