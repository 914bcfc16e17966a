// Text-query attention over [visual; text] keys on gfx950 (Section 3.2, Eq. 9).
//
// Every text query reads all Nv visual keys of its kv-head and the text keys up
// to its own position (visual tokens precede the text, Section 2 Eq. 2).
//
//   k_attn_prefill  MFMA flash attention. Query rows of one kv-head group are
//                   packed (row = query * G + head-in-group) so GQA heads share
//                   each K/V tile. Scores are formed transposed, S^T = K Q^T,
//                   and the output as O^T = V^T P^T: the accumulator layout then
//                   keeps one query per lane, so the running max / sum and the
//                   rescale of O are per-lane and P feeds the second product
//                   straight from registers. K/V tiles stream through padded
//                   LDS rows (conflict-free for both access patterns).
//   k_attn_decode   one query per sequence: a bandwidth-bound stream over the
//                   K/V caches with 16-byte loads, dot products reduced across
//                   the lanes of one key row, and an online softmax.
//   k_attn_stream   bf16, hd 128 prefill: the same math with K/V tiles loaded straight into
//                   LDS (range-checked buffer loads, two stages in flight), keys walked as
//                   visual tiles then text tiles so each tile has one source, and the V^T
//                   fragment read with two ds_read_b64_tr_b16 transpose loads.
//   k_attn_combine  log-sum-exp merge of key-split partials.
#include "attention.hpp"
#include "dv_device.hpp"
#include "gemm_pipe.hpp"

#include <math.h>

#include <mutex>
#include <type_traits>

#include "../../include/deltavision.h"

namespace dv {

constexpr float NEG_BIG = -1e30f;  // finite start value of the running max

__device__ __forceinline__ u32x4 ld16(const void* p) { return *(const u32x4*)p; }
// Non-temporal 16-byte load, for data read once.
__device__ __forceinline__ u32x4 ld16_stream(const void* p) {
  return __builtin_nontemporal_load((const u32x4*)p);
}

template <typename T, int HD, int NW>
struct AttnCfg {
  static constexpr int NKB = sizeof(T) == 2 ? 2 : 1;  // 32-key sub-tiles per tile
  static constexpr int KT = 32 * NKB;              // keys per tile (LDS stays below 64 KiB)
  static constexpr int NT = NW * WAVE;
  static constexpr int EPC = 16 / (int)sizeof(T);  // elements per 16-byte chunk
  static constexpr int PITCH = HD + EPC;           // LDS row pitch: 16-byte pad per row
  static constexpr int CPR = HD / EPC;             // chunks per K/V row
  static constexpr int LD_IT = KT * CPR / NT;      // chunks per thread per tile and tensor
  static constexpr int KS = HD / 16;               // 16-deep K steps of S^T = K Q^T
  static constexpr int CB = HD / 32;               // 32-row blocks of O^T
  static constexpr int LDS_BYTES = 2 * KT * PITCH * (int)sizeof(T);
  static_assert((KT * CPR) % NT == 0, "tile chunks must divide threads");
};

template <typename T>
__device__ __forceinline__ typename Frag8<T>::type lds_row8(const T* s);
template <>
__device__ __forceinline__ bf16x8 lds_row8<bf16>(const bf16* s) {
  return __builtin_bit_cast(bf16x8, ld16(s));
}
template <>
__device__ __forceinline__ f32x8 lds_row8<float>(const float* s) {
  f32x4 a = __builtin_bit_cast(f32x4, ld16(s)), b = __builtin_bit_cast(f32x4, ld16(s + 4));
  return f32x8{a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
}

template <typename T>
__device__ __forceinline__ void load_row8_f32(const T* p, float (&x)[8]);
template <>
__device__ __forceinline__ void load_row8_f32<bf16>(const bf16* p, float (&x)[8]) {
  bf16x8 v = __builtin_bit_cast(bf16x8, ld16(p));
#pragma unroll
  for (int e = 0; e < 8; ++e) x[e] = (float)v[e];
}
template <>
__device__ __forceinline__ void load_row8_f32<float>(const float* p, float (&x)[8]) {
  f32x4 a = __builtin_bit_cast(f32x4, ld16(p)), b = __builtin_bit_cast(f32x4, ld16(p + 4));
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    x[e] = a[e];
    x[4 + e] = b[e];
  }
}

template <typename T>
__device__ __forceinline__ void store4(T* p, float a, float b, float c, float d);
template <>
__device__ __forceinline__ void store4<bf16>(bf16* p, float a, float b, float c, float d) {
  bf16x4 v = {(bf16)a, (bf16)b, (bf16)c, (bf16)d};
  *(u32x2*)p = __builtin_bit_cast(u32x2, v);
}
template <>
__device__ __forceinline__ void store4<float>(float* p, float a, float b, float c, float d) {
  *(f32x4*)p = f32x4{a, b, c, d};
}

// ------------------------------------------------------------------ prefill

template <typename T, int HD, int NW>
__global__ __launch_bounds__(NW * 64) void k_attn_prefill(AttnArgs a) {
  typedef AttnCfg<T, HD, NW> C;
  typedef typename Frag8<T>::type Fr;
  extern __shared__ __align__(16) unsigned char smem[];
  T* sk = (T*)smem;
  T* sv = sk + C::KT * C::PITCH;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, g2 = lane >> 5;
  const int G = a.Hq / a.Hkv, R = a.Nq * G;
  const int bg = blockIdx.y, b = bg / a.Hkv, g = bg - b * a.Hkv;
  const int split = blockIdx.z;

  // Rows of this block / wave. Row r <-> query i = r / G, head h = g*G + r % G.
  const int row0 = blockIdx.x * (32 * NW);
  const int my_row = row0 + wave * 32 + (lane & 31);
  const bool row_ok = my_row < R;
  const int my_i = row_ok ? my_row / G : 0;
  const int my_h = g * G + (row_ok ? my_row - my_i * G : 0);
  const int last_row = min(row0 + 32 * NW, R) - 1;
  const int i_max = last_row / G;

  // Key range: this split's slice of [visual; text] cut at the furthest causal limit.
  const int nk_all = a.Nv + a.q_pos0 + i_max + 1;
  const int k_begin = split * a.keys_per_split;
  const int k_end = min(nk_all, k_begin + a.keys_per_split);

  const T* Kvb = (const T*)a.Kv + (int64_t)bg * a.Nv * HD;
  const T* Vvb = (const T*)a.Vv + (int64_t)bg * a.Nv * HD;
  const T* Ktb = (const T*)a.Kt + (int64_t)bg * a.Nkt * HD;
  const T* Vtb = (const T*)a.Vt + (int64_t)bg * a.Nkt * HD;

  // Q^T fragments of this lane's row (B operand), pre-scaled by scale*log2(e).
  Fr qf[C::KS];
  {
    const T* qrow = (const T*)a.Q + (((int64_t)b * a.Nq + my_i) * a.Hq + my_h) * HD;
#pragma unroll
    for (int ks = 0; ks < C::KS; ++ks) {
      float x[8];
      if (row_ok) load_row8_f32<T>(qrow + ks * 16 + g2 * 8, x);
#pragma unroll
      for (int e = 0; e < 8; ++e) qf[ks][e] = from_f32<T>(row_ok ? x[e] : 0.f);
    }
  }
  const float qscale = a.scale_log2;

  f32x16 oacc[C::CB];
#pragma unroll
  for (int cb = 0; cb < C::CB; ++cb) oacc[cb] = f32x16{};
  float m_run = NEG_BIG, l_run = 0.f;
  const int my_text_lim = a.Nv + a.q_pos0 + my_i;  // last allowed key index for my row

  u32x4 rk[C::LD_IT], rv[C::LD_IT];
  auto gload = [&](int k0) {
#pragma unroll
    for (int it = 0; it < C::LD_IT; ++it) {
      const int idx = tid + it * C::NT, key = idx / C::CPR, ch = idx - key * C::CPR;
      const int j = k0 + key;
      if (j < k_end) {
        const T* ks_ = j < a.Nv ? Kvb + (int64_t)j * HD : Ktb + (int64_t)(j - a.Nv) * HD;
        const T* vs_ = j < a.Nv ? Vvb + (int64_t)j * HD : Vtb + (int64_t)(j - a.Nv) * HD;
        rk[it] = ld16(ks_ + ch * C::EPC);
        rv[it] = ld16(vs_ + ch * C::EPC);
      } else {
        rk[it] = u32x4{0, 0, 0, 0};
        rv[it] = u32x4{0, 0, 0, 0};
      }
    }
  };
  auto sstore = [&]() {
#pragma unroll
    for (int it = 0; it < C::LD_IT; ++it) {
      const int idx = tid + it * C::NT, key = idx / C::CPR, ch = idx - key * C::CPR;
      *(u32x4*)(sk + key * C::PITCH + ch * C::EPC) = rk[it];
      *(u32x4*)(sv + key * C::PITCH + ch * C::EPC) = rv[it];
    }
  };

  if (k_begin < k_end) gload(k_begin);
  for (int k0 = k_begin; k0 < k_end; k0 += C::KT) {
    __syncthreads();  // previous tile fully consumed
    sstore();
    __syncthreads();
    if (k0 + C::KT < k_end) gload(k0 + C::KT);

    // S^T (keys x my queries), one accumulator per 32-key sub-tile.
    f32x16 sacc[C::NKB];
#pragma unroll
    for (int kb = 0; kb < C::NKB; ++kb) {
      sacc[kb] = f32x16{};
#pragma unroll
      for (int ks = 0; ks < C::KS; ++ks) {
        Fr kf = lds_row8<T>(sk + (kb * 32 + (lane & 31)) * C::PITCH + ks * 16 + g2 * 8);
        mfma_k16(sacc[kb], kf, qf[ks]);
      }
    }
    // Mask, scale and the running max of my query (shared by the two lane halves).
    float tmax = NEG_BIG;
#pragma unroll
    for (int kb = 0; kb < C::NKB; ++kb)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const int j = k0 + kb * 32 + acc_row(lane, i);
        const bool ok = j < k_end && j <= my_text_lim;
        const float s = ok ? sacc[kb][i] * qscale : -INFINITY;
        sacc[kb][i] = s;
        tmax = fmaxf(tmax, s);
      }
    tmax = fmaxf(tmax, shfl_xor(tmax, 32));
    const float m_new = fmaxf(m_run, tmax);
    const float alpha = exp2f(m_run - m_new);
    m_run = m_new;
    float psum = 0.f;
#pragma unroll
    for (int kb = 0; kb < C::NKB; ++kb)
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        const float p = exp2f(sacc[kb][i] - m_new);
        sacc[kb][i] = p;
        psum += p;
      }
    l_run = l_run * alpha + psum;
#pragma unroll
    for (int cb = 0; cb < C::CB; ++cb) oacc[cb] *= alpha;

    // O^T += V^T P^T. P^T item i of sub-tile kb is key kb*32 + acc_row(lane, i); the
    // 16-deep K step s2 takes items 8*s2..8*s2+7, so V^T slot e of lane half g2 is key
    // kb*32 + 16*s2 + (e/4)*8 + 4*g2 + e%4.
#pragma unroll
    for (int kb = 0; kb < C::NKB; ++kb) {
#pragma unroll
      for (int s2 = 0; s2 < 2; ++s2) {
        Fr pf;
#pragma unroll
        for (int e = 0; e < 8; ++e) pf[e] = from_f32<T>(sacc[kb][s2 * 8 + e]);
        const int kbase = kb * 32 + 16 * s2 + 4 * g2;
#pragma unroll
        for (int cb = 0; cb < C::CB; ++cb) {
          const T* vcol = sv + cb * 32 + (lane & 31);
          Fr vf;
#pragma unroll
          for (int e = 0; e < 8; ++e) vf[e] = vcol[(kbase + (e >> 2) * 8 + (e & 3)) * C::PITCH];
          mfma_k16(oacc[cb], vf, pf);
        }
      }
    }
  }

  const float l_tot = l_run + shfl_xor(l_run, 32);
  if (!row_ok) return;
  const int64_t orow = ((int64_t)b * a.Nq + my_i) * a.Hq + my_h;
  if (a.splits == 1) {
    const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
    T* o = (T*)a.O + orow * HD;
#pragma unroll
    for (int cb = 0; cb < C::CB; ++cb)
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        const int c = cb * 32 + q4 * 8 + g2 * 4;
        store4<T>(o + c, oacc[cb][q4 * 4] * inv, oacc[cb][q4 * 4 + 1] * inv,
                  oacc[cb][q4 * 4 + 2] * inv, oacc[cb][q4 * 4 + 3] * inv);
      }
  } else {
    const int64_t rows_total = (int64_t)a.B * a.Nq * a.Hq;
    float* op = a.Opart + ((int64_t)split * rows_total + orow) * HD;
#pragma unroll
    for (int cb = 0; cb < C::CB; ++cb)
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        const int c = cb * 32 + q4 * 8 + g2 * 4;
        *(f32x4*)(op + c) = f32x4{oacc[cb][q4 * 4], oacc[cb][q4 * 4 + 1], oacc[cb][q4 * 4 + 2],
                                  oacc[cb][q4 * 4 + 3]};
      }
    if (g2 == 0) {
      float* ml = a.MLpart + ((int64_t)split * rows_total + orow) * 2;
      ml[0] = m_run;
      ml[1] = l_tot;
    }
  }
}


// ------------------------------------------------------------------ streaming prefill (bf16)

namespace stream {
constexpr int HD = 128;
constexpr int KT = 64;                    // keys per tile
constexpr int ROWB = HD * 2;              // bytes per K/V row
constexpr int TILE_BYTES = KT * ROWB;     // one tensor's tile: 16 KiB
constexpr int STAGE_BYTES = 2 * TILE_BYTES;
// Stages: up to two tiles keep loading while one is computed. A wave counts at most 63
// outstanding loads (6-bit vmcnt), i.e. two tiles of a single-wave block. The streaming kernel
// runs with two waves (65 to 96 rows per kv-head); more rows go to the ping-pong kernel below.
template <int NW> constexpr int stages() { return NW == 4 ? 2 : 3; }
// Streaming blocks that fit in one CU's 160 KiB of LDS.
template <int NW> constexpr int blocks_per_cu() { return (160 * 1024) / (stages<NW>() * 2 * 64 * 256); }
template <int NW> constexpr int lds_bytes() { return stages<NW>() * STAGE_BYTES; }
// Cache-policy bits of the tile loads. A K/V tile that only one block reads is loaded
// non-temporally (LLaVA-NeXT, 128 rows per kv-head: 91.5 -> 81 us per layer with the four-wave
// streaming kernel); tiles that several row blocks share keep the default policy, so the later
// readers still find them in the L2 (Qwen2.5-VL video, seven row blocks: non-temporal loads
// cost about 1.5%).
constexpr int CPOL_DEFAULT = 0;
constexpr int CPOL_NT = 2;
constexpr int BLOCKS_PER_TILE = KT / 4;   // 1 KiB (4-row) load instructions per tensor
// XOR keys of the 16-byte chunks of a 256-byte LDS row. K rows are read whole-chunk by 16 rows
// at once (key = row mod 16). V rows are read by the transpose loads, whose 32-lane halves each
// take 4 consecutive rows x 4 consecutive chunks (two column blocks of 16 lanes): key =
// 4 * (row mod 4) gives each of the 4 rows its own quarter of the 64 banks. (A key of
// 2 * (row mod 8), which separates the 16 lanes of one column block only, measured about one
// conflict cycle per LDS instruction; this key measures none.)
__device__ __forceinline__ int key_k(int row) { return row & 15; }
__device__ __forceinline__ int key_v(int row) { return (row & 3) << 2; }
}  // namespace stream

typedef short s16x4 __attribute__((ext_vector_type(4)));

// Transposed LDS reads of V (ds_read_b64_tr_b16) issued as inline assembly. The compiler's
// wait-count pass cannot tell an LDS read from the direct-to-LDS loads still in flight into the
// other stages (one dynamic LDS object), so before every such read it can see it drains all of
// them (vmcnt(0)), which leaves the next tiles' loads half a tile instead of a whole one to land.
// The kernels' own waits already make each stage's loads land before it is read. A read's
// result is used only after lds_wait(), whose assembly waits for every LDS read and ties the
// result registers, so no use can be scheduled before it.
// The LDS address is a per-lane base plus the constant OFF (the instruction's offset field).
template <int OFF>
__device__ __forceinline__ s16x4 lds_read_tr16(uint32_t base) {
  static_assert(OFF >= 0 && OFF < 65536, "16-bit LDS offset");
  s16x4 r;
  asm volatile("ds_read_b64_tr_b16 %0, %1 offset:%2" : "=v"(r) : "v"(base), "n"(OFF));
  return r;
}
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
}
// V^T fragments of one 16-key step (keys KEY0 .. KEY0 + 15 of the stage's tile) for the four
// 32-column blocks: col[cb] is the lane's address of key row vrow (< 8) of column block cb
// relative to the stage (rows a multiple of 4 apart share the chunk swizzle, so every read of a
// lane differs only by a constant); the two reads per block return slots 0..3 and 4..7.
template <int ROWB, int KEY0>
__device__ __forceinline__ void read_v_step(uint32_t stage, const uint32_t (&col)[4],
                                            s16x4 (&vr)[8]) {
#pragma unroll
  for (int cb = 0; cb < 4; ++cb) {
    vr[2 * cb] = lds_read_tr16<KEY0 * ROWB>(stage + col[cb]);
    vr[2 * cb + 1] = lds_read_tr16<(KEY0 + 8) * ROWB>(stage + col[cb]);
  }
}
// LEFT: how many of the most recently issued LDS (or scalar) operations may stay outstanding;
// LDS operations complete in issue order, so every earlier LDS read has returned.
template <int LEFT = 0, int N>
__device__ __forceinline__ void lds_wait(s16x4 (&v)[N]) {
  static_assert(LEFT >= 0 && LEFT <= 15, "lgkmcnt counts up to 15");
  asm volatile("s_waitcnt lgkmcnt(%0)" ::"n"(LEFT));
#pragma unroll
  for (int i = 0; i < N; ++i) asm volatile("" : "+v"(v[i]));
}

// Online-softmax step of one tile for the query row of this lane (the two lane halves hold the
// same row). Scores arrive raw; masked ones are -inf; they leave as p = 2^(s*scale - m). The
// running max m (in units of scale*log2 e) is only raised when some row of the wave grew by more
// than 2^8: between raises p stays below 256, and since the sum and O use the same stale m the
// result is unchanged while most tiles skip the rescale of O. The caller adds the tile's p to
// the row sum l_run (after rounding them for the P V product, see add_probs).
// The scores are the MFMA accumulator tiles themselves, worked on in place (a copy into a plain
// array cost one move per score: the masking branch made the compiler keep both).
template <int NB, int NCB>
__device__ __forceinline__ void online_softmax(f32x16 (&sv)[NB], float scale_log2, float& m_run,
                                               float& l_run, f32x16 (&oacc)[NCB]) {
  float tmax = -INFINITY;
#pragma unroll
  for (int b = 0; b < NB; ++b)
#pragma unroll
    for (int i = 0; i < 16; ++i) tmax = fmaxf(tmax, sv[b][i]);
  tmax = fmaxf(tmax, shfl_xor(tmax, 32)) * scale_log2;
  const bool grow = tmax > m_run + 8.0f;
  if (__builtin_amdgcn_ballot_w64(grow) != 0) {
    const float m_new = fmaxf(m_run, tmax);
    const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
    m_run = m_new;
    l_run *= alpha;
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) oacc[cb] *= alpha;
  }
  const float neg_m = -m_run;
#pragma unroll
  for (int b = 0; b < NB; ++b)
#pragma unroll
    for (int i = 0; i < 16; ++i)
      sv[b][i] = __builtin_amdgcn_exp2f(fmaf(sv[b][i], scale_log2, neg_m));
}

// Adds the eight bf16 probabilities of a P fragment to a row sum: the sum is taken over the
// same rounded values that the P V product multiplies, two per dot-product instruction.
__device__ __forceinline__ float add_probs(const bf16x8& p, float sum) {
  typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
  const bf16x2 one = {(bf16)1.0f, (bf16)1.0f};
#pragma unroll
  for (int q = 0; q < 4; ++q)
    sum = __builtin_amdgcn_fdot2_f32_bf16(bf16x2{p[2 * q], p[2 * q + 1]}, one, sum, false);
  return sum;
}

// Block-uniform integer that the compiler computes on the vector unit (integer divisions):
// stating it is uniform keeps load bases and sizes in scalar registers.
__device__ __forceinline__ int uni(int x) { return __builtin_amdgcn_readfirstlane(x); }

// Work of a prefill block: (batch * kv-head group bg, block of query rows rb, key split). The
// dispatcher deals consecutive launch ids out to the 8 XCDs in turn, so ids congruent mod 8 run on
// one XCD. All row blocks of one (bg, split) stream read the same K/V range: they get ids x,
// x + 8, x + 16, ..., so that range comes from memory once into that XCD's L2. Streams left over
// when their count is not a multiple of 8 are laid out contiguously.
struct BlockWork {
  int bg, rb, split;
};
__device__ __forceinline__ BlockWork block_work(int n_bg, int row_blocks, int splits) {
  const int id = blockIdx.x + gridDim.x * blockIdx.y;
  const int streams = n_bg * splits, full = (streams / 8) * 8 * row_blocks;
  int s, rb;
  if (id < full) {
    const int slot = id / 8;
    rb = slot % row_blocks;
    s = (slot / row_blocks) * 8 + id % 8;
  } else {
    const int r = id - full;
    rb = r % row_blocks;
    s = (streams / 8) * 8 + r / row_blocks;
  }
  return BlockWork{uni(s / splits), uni(rb), uni(s % splits)};
}

// Wait until tile t+1 of the pipeline has landed when `ahead` later tiles may stay in flight
// (never encoding more than the 63 loads vmcnt can count), then synchronise the block.
template <int INS>
__device__ __forceinline__ void stream_sync(int ahead) {
  constexpr int kMaxTiles = 63 / INS;
  if (ahead > kMaxTiles) ahead = kMaxTiles;
  if (ahead >= 2) pipe_sync<waitcnt_imm((kMaxTiles >= 2 ? 2 : 0) * INS, 0)>();
  else if (ahead == 1) pipe_sync<waitcnt_imm(INS, 0)>();
  else pipe_sync<waitcnt_imm(0, 0)>();
}

template <int NW, int CPOL>
__global__ __launch_bounds__(NW * 64, NW == 4 ? 2 : 1) void k_attn_stream(AttnArgs a, int row_blocks) {
  using namespace stream;
  constexpr int NS = stages<NW>();
  constexpr int INS = 2 * BLOCKS_PER_TILE / NW;  // load instructions per wave per tile
  static_assert(NS - 1 <= 2 && INS <= 63, "stream_sync handles at most two tiles in flight");
  static_assert(BLOCKS_PER_TILE % NW == 0, "waves must split the tile loads evenly");
  extern __shared__ __align__(16) unsigned char smem[];

  const int lane = threadIdx.x & 63, wave = wave_index(), g2 = lane >> 5;
  const int G = a.Hq / a.Hkv, R = a.Nq * G, n_bg = a.B * a.Hkv;

  const BlockWork wk = block_work(n_bg, row_blocks, a.splits);
  const int rb = wk.rb, bg = wk.bg, split = wk.split;
  const int b = uni(bg / a.Hkv), g = bg - b * a.Hkv;
  const int row0 = rb * 32 * NW;
  const int my_row = row0 + wave * 32 + (lane & 31);
  const bool row_ok = my_row < R;
  const int my_i = row_ok ? my_row / G : 0;
  const int my_h = g * G + (row_ok ? my_row - my_i * G : 0);
  const int i_max = uni((min(row0 + 32 * NW, R) - 1) / G);
  const int text_lim = min(a.Nkt, a.q_pos0 + i_max + 1);  // text keys any row of the block needs
  const int my_text_last = a.q_pos0 + my_i;                // last text key of my row
  const int tv = uni((a.Nv + KT - 1) / KT), ntiles = uni(tv + (text_lim + KT - 1) / KT);
  const int t_begin = split * a.tiles_per_split;
  const int t_end = min(ntiles, t_begin + a.tiles_per_split);

  const bf16* kvb = (const bf16*)a.Kv + (int64_t)bg * a.Nv * HD;
  const bf16* vvb = (const bf16*)a.Vv + (int64_t)bg * a.Nv * HD;
  const bf16* ktb = (const bf16*)a.Kt + (int64_t)bg * a.Nkt * HD;
  const bf16* vtb = (const bf16*)a.Vt + (int64_t)bg * a.Nkt * HD;
  const int64_t vis_bytes = (int64_t)a.Nv * ROWB, txt_bytes = (int64_t)text_lim * ROWB;

  // Q^T fragments of my row (B operand of S^T = K Q^T).
  bf16x8 qf[HD / 16];
  {
    const bf16* qrow = (const bf16*)a.Q + (((int64_t)b * a.Nq + my_i) * a.Hq + my_h) * HD;
#pragma unroll
    for (int ks = 0; ks < HD / 16; ++ks)
      qf[ks] = row_ok ? __builtin_bit_cast(bf16x8, ld16(qrow + ks * 16 + g2 * 8)) : bf16x8{};
  }

  // Lane part of a load instruction: row r4 = lane / 16 of a 4-row block, LDS chunk pc.
  const int r4 = lane >> 4, pc = lane & 15;
  auto issue = [&](int t, int stage) {
    const bool vis = t < tv;
    const int key0 = (vis ? t : t - tv) * KT;
    unsigned char* sk = smem + stage * STAGE_BYTES;
    unsigned char* sv = sk + TILE_BYTES;
    // Select the (uniform) base and size, then build the resources: a select between two
    // resources would be lowered per lane and force a waterfall loop around every load.
    const __amdgpu_buffer_rsrc_t rk = buffer_rsrc(vis ? kvb : ktb, vis ? vis_bytes : txt_bytes);
    const __amdgpu_buffer_rsrc_t rv = buffer_rsrc(vis ? vvb : vtb, vis ? vis_bytes : txt_bytes);
#pragma unroll
    for (int i = 0; i < BLOCKS_PER_TILE / NW; ++i) {
      const int blk = wave * (BLOCKS_PER_TILE / NW) + i;
      const int row = blk * 4 + r4;
      const int soff = (key0 + blk * 4) * ROWB;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rk, (lds_void*)(sk + blk * 1024), 16,
                                               r4 * ROWB + ((pc ^ key_k(row)) << 4), soff, 0, CPOL);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rv, (lds_void*)(sv + blk * 1024), 16,
                                               r4 * ROWB + ((pc ^ key_v(row)) << 4), soff, 0, CPOL);
    }
  };

  f32x16 oacc[HD / 32];
#pragma unroll
  for (int cb = 0; cb < HD / 32; ++cb) oacc[cb] = f32x16{};
  float m_run = NEG_BIG, l_run = 0.f;

  // Prologue: fill every stage, then wait for the first tile only.
  const int nt = t_end - t_begin;
#pragma unroll
  for (int j = 0; j < NS; ++j)
    if (j < nt) issue(t_begin + j, j);
  stream_sync<INS>(min(NS, nt) - 1);

  // Transpose-load lane roles (fixed for the whole loop): in each 16-lane group, lane L points
  // at key row (L / 4) of a 4-key group and columns c0 + 4 (L % 4) .. + 3 of it.
  const int l16 = lane & 15, grp = lane >> 4;
  const int tr_row = l16 >> 2;
  const int tr_col = 16 * (grp & 1) + 4 * (l16 & 3);  // plus 32 * cb
  // V read addresses inside a stage's V tile: key row vrow of the step, column block cb.
  uint32_t vcol[4];
  {
    const int vrow = 4 * (grp >> 1) + tr_row;
#pragma unroll
    for (int cb = 0; cb < 4; ++cb) {
      const int col = 32 * cb + tr_col;
      vcol[cb] = vrow * ROWB + (((col >> 3) ^ key_v(vrow)) << 4) + (col & 7) * 2;
    }
  }

  int stage = 0;
  for (int t = t_begin; t < t_end; ++t) {
    const unsigned char* sk = smem + stage * STAGE_BYTES;
    const unsigned char* sv = sk + TILE_BYTES;
    const bool vis = t < tv;
    const int key0 = (vis ? t : t - tv) * KT;

    f32x16 sacc[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      sacc[kb] = f32x16{};
      const int row = kb * 32 + (lane & 31);
#pragma unroll
      for (int ks = 0; ks < HD / 16; ++ks) {
        const int chunk = ks * 2 + g2;
        bf16x8 kf = __builtin_bit_cast(
            bf16x8, *(const u32x4*)(sk + row * ROWB + ((chunk ^ key_k(row)) << 4)));
        mfma_k16(sacc[kb], kf, qf[ks]);
      }
    }
    if (!vis || key0 + KT > a.Nv) {  // partial visual tile or text tile: mask
      // The last key of this tile's kind the lane's row sees, relative to the tile: one compare
      // and select per score.
      const int last = (vis ? a.Nv - 1 : min(my_text_last, text_lim - 1)) - key0;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int i = 0; i < 16; ++i)
          sacc[kb][i] = kb * 32 + acc_row(lane, i) > last ? -INFINITY : sacc[kb][i];
    }
    online_softmax(sacc, a.scale_log2, m_run, l_run, oacc);

    // O^T += V^T P^T. For K step (kb, s2) slot e of lane half g2 is key
    // kb*32 + 16*s2 + (e/4)*8 + 4*g2 + e%4 in both operands; the two transpose loads return
    // slots 0..3 and 4..7 of V^T for column 32*cb + lane % 32. All 32 reads of the tile go out
    // together; the first key block's 16 are waited for before its MFMAs, the rest after them.
    s16x4 vbuf[4][2 * (HD / 32)];
    float lsum[2] = {0.f, 0.f};  // two chains of the tile's row sum
    const uint32_t vs = lds_addr(sv);
    read_v_step<ROWB, 0>(vs, vcol, vbuf[0]);
    read_v_step<ROWB, 16>(vs, vcol, vbuf[1]);
    read_v_step<ROWB, 32>(vs, vcol, vbuf[2]);
    read_v_step<ROWB, 48>(vs, vcol, vbuf[3]);
#pragma unroll
    for (int step = 0; step < 4; ++step) {
      if (step == 0) {
        // At most 15 of the 32 still out: the first 16 (key block 0) have returned.
        lds_wait<15>(vbuf[0]);
        lds_wait<15>(vbuf[1]);
      } else if (step == 2) {
        lds_wait(vbuf[2]);
        lds_wait(vbuf[3]);
      }
      const int kb = step >> 1, s2 = step & 1;
      bf16x8 pf;
#pragma unroll
      for (int e = 0; e < 8; ++e) pf[e] = (bf16)sacc[kb][s2 * 8 + e];
      lsum[s2] = add_probs(pf, lsum[s2]);
#pragma unroll
      for (int cb = 0; cb < HD / 32; ++cb) {
        const s16x4 vv[2] = {vbuf[step][2 * cb], vbuf[step][2 * cb + 1]};
        mfma_k16(oacc[cb], __builtin_bit_cast(bf16x8, vv), pf);
      }
    }
    l_run += lsum[0] + lsum[1];

    // Tile t+1 has landed (tiles t+2 .. t+NS-1 may still load) and every wave is done with
    // this stage: refill it with tile t+NS.
    stream_sync<INS>(min(NS - 2, t_end - t - 2));
    if (t + NS < t_end) issue(t + NS, stage);
    stage = stage + 1 == NS ? 0 : stage + 1;
  }

  const float l_tot = l_run + shfl_xor(l_run, 32);
  if (!row_ok) return;
  const int64_t orow = ((int64_t)b * a.Nq + my_i) * a.Hq + my_h;
  if (a.splits == 1) {
    const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
    bf16* o = (bf16*)a.O + orow * HD;
#pragma unroll
    for (int cb = 0; cb < HD / 32; ++cb)
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        const int c = cb * 32 + q4 * 8 + g2 * 4;
        store4<bf16>(o + c, oacc[cb][q4 * 4] * inv, oacc[cb][q4 * 4 + 1] * inv,
                     oacc[cb][q4 * 4 + 2] * inv, oacc[cb][q4 * 4 + 3] * inv);
      }
  } else {
    const int64_t rows_total = (int64_t)a.B * a.Nq * a.Hq;
    float* op = a.Opart + ((int64_t)split * rows_total + orow) * HD;
#pragma unroll
    for (int cb = 0; cb < HD / 32; ++cb)
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        const int c = cb * 32 + q4 * 8 + g2 * 4;
        *(f32x4*)(op + c) = f32x4{oacc[cb][q4 * 4], oacc[cb][q4 * 4 + 1], oacc[cb][q4 * 4 + 2],
                                  oacc[cb][q4 * 4 + 3]};
      }
    if (g2 == 0) {
      float* ml = a.MLpart + ((int64_t)split * rows_total + orow) * 2;
      ml[0] = m_run;
      ml[1] = l_tot;
    }
  }
}

// ------------------------------------------------------------------ ping-pong streaming prefill
//
// Many rows per kv-head (bf16, hd 128): a block of eight waves takes 128 (query, GQA-head) rows.
// Waves w and w + 4 hold the same 32 rows; the first group of four takes the even key tiles of
// the block's range, the second the odd ones, and the two partial (max, sum, O) of a row merge
// through LDS at the end. A group works in alternating phases separated by block barriers: an
// MFMA phase (P V of its previous tile, then the scores of its next tile) and a softmax phase
// (the VALU work of that tile's probabilities). The second group runs one phase behind the first,
// so on every SIMD one wave issues MFMAs while the other works on the VALU: the dependency chain
// scores -> softmax -> P V of one tile no longer leaves the matrix pipe idle.
// Each group streams its K tiles and V tiles through rings of two slots; a K tile is read in the
// MFMA phase that forms its scores and a V tile one MFMA phase later, so every refill has two
// phases to land. Tiles past the end of a group's share come from an empty buffer range (the
// loads return zeros without touching memory), so every wave issues the same loads in every
// phase and one constant wait count holds throughout.
namespace pp {
constexpr int HD = 128;
constexpr int KT = 64;                      // keys per tile
constexpr int ROWB = HD * 2;
constexpr int TILE_BYTES = KT * ROWB;       // one tensor's tile: 16 KiB
constexpr int NRW = 4;                      // waves per group, 32 rows each
constexpr int NWAVE = 2 * NRW;
constexpr int GROUP_BYTES = 4 * TILE_BYTES; // two K slots, two V slots
constexpr int LDS_BYTES = 2 * GROUP_BYTES;  // 128 KiB; the merge reuses it
constexpr int LD = TILE_BYTES / 1024 / NRW; // 1 KiB loads per wave per tensor tile
constexpr int MPITCH = HD + 4;              // merge rows padded by 16 B
static_assert(NRW * 32 * (MPITCH + 2) * 4 <= LDS_BYTES, "merge buffer must fit");
static_assert(2 * LD <= 63, "vmcnt counts every load in flight");
}  // namespace pp

template <int CPOL>
__global__ __launch_bounds__(pp::NWAVE * 64, 1) void k_attn_pp(AttnArgs a, int row_blocks) {
  using namespace pp;
  extern __shared__ __align__(16) unsigned char smem[];

  const int lane = threadIdx.x & 63, wave = wave_index(), g2 = lane >> 5;
  const int grp = uni(wave / NRW), rw = uni(wave % NRW);
  const int G = a.Hq / a.Hkv, R = a.Nq * G, n_bg = a.B * a.Hkv;

  const BlockWork wk = block_work(n_bg, row_blocks, a.splits);
  const int rb = wk.rb, bg = wk.bg, split = wk.split;
  const int b = uni(bg / a.Hkv), g = bg - b * a.Hkv;
  const int row0 = rb * 32 * NRW;
  const int my_row = row0 + rw * 32 + (lane & 31);
  const bool row_ok = my_row < R;
  const int my_i = row_ok ? my_row / G : 0;
  const int my_h = g * G + (row_ok ? my_row - my_i * G : 0);
  const int i_max = uni((min(row0 + 32 * NRW, R) - 1) / G);
  const int text_lim = min(a.Nkt, a.q_pos0 + i_max + 1);  // text keys any row of the block needs
  const int my_text_last = a.q_pos0 + my_i;                // last text key of my row
  const int tv = uni((a.Nv + KT - 1) / KT), ntiles = uni(tv + (text_lim + KT - 1) / KT);
  const int t_begin = split * a.tiles_per_split;
  const int t_end = min(ntiles, t_begin + a.tiles_per_split);
  const int n = max(0, t_end - t_begin);
  const int nA = (n + 1) / 2, nB = n / 2;
  const int nj = grp == 0 ? nA : nB;                     // my group's tiles: t_begin + grp + 2 j

  const bf16* kvb = (const bf16*)a.Kv + (int64_t)bg * a.Nv * HD;
  const bf16* vvb = (const bf16*)a.Vv + (int64_t)bg * a.Nv * HD;
  const bf16* ktb = (const bf16*)a.Kt + (int64_t)bg * a.Nkt * HD;
  const bf16* vtb = (const bf16*)a.Vt + (int64_t)bg * a.Nkt * HD;
  const int64_t vis_bytes = (int64_t)a.Nv * ROWB, txt_bytes = (int64_t)text_lim * ROWB;

  bf16x8 qf[HD / 16];
  {
    const bf16* qrow = (const bf16*)a.Q + (((int64_t)b * a.Nq + my_i) * a.Hq + my_h) * HD;
#pragma unroll
    for (int ks = 0; ks < HD / 16; ++ks)
      qf[ks] = row_ok ? __builtin_bit_cast(bf16x8, ld16(qrow + ks * 16 + g2 * 8)) : bf16x8{};
  }

  unsigned char* gbase = smem + grp * GROUP_BYTES;
  const int r4 = lane >> 4, pc = lane & 15;
  // This wave's quarter (4 of the 16 four-row blocks) of K or V of my group's tile j, into ring
  // slot j % 2. The base and size are selected first (uniform), then the resource is built.
  auto issue = [&](int j, auto is_v) {
    constexpr bool V = decltype(is_v)::value;
    const int t = t_begin + grp + 2 * j;
    const bool in = j < nj;
    const bool vis = t < tv;
    const int key0 = in ? (vis ? t : t - tv) * KT : 0;
    const bf16* base = vis ? (V ? vvb : kvb) : (V ? vtb : ktb);
    const int64_t bytes = in ? (vis ? vis_bytes : txt_bytes) : 0;
    const __amdgpu_buffer_rsrc_t rs = buffer_rsrc(base, bytes);
    unsigned char* dst = gbase + (V ? 2 * TILE_BYTES : 0) + (j & 1) * TILE_BYTES;
#pragma unroll
    for (int i = 0; i < LD; ++i) {
      const int blk = rw * LD + i;
      const int row = blk * 4 + r4;
      const int key = V ? stream::key_v(row) : stream::key_k(row);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_void*)(dst + blk * 1024), 16,
                                               r4 * ROWB + ((pc ^ key) << 4),
                                               (key0 + blk * 4) * ROWB, 0, CPOL);
    }
  };
  using KTag = std::integral_constant<bool, false>;
  using VTag = std::integral_constant<bool, true>;
  // Prologue, oldest first: K of tile 0, then what the steady state issues after MFMA phase k
  // (K of tile k + 2, V of tile k + 1) for k = -1.
  issue(0, KTag{});
  issue(1, KTag{});
  issue(0, VTag{});

  const int l16 = lane & 15, grp16 = lane >> 4;
  const int tr_row = l16 >> 2;
  const int tr_col = 16 * (grp16 & 1) + 4 * (l16 & 3);
  uint32_t vcol[4];  // as in k_attn_stream
  {
    const int vrow = 4 * (grp16 >> 1) + tr_row;
#pragma unroll
    for (int cb = 0; cb < 4; ++cb) {
      const int col = 32 * cb + tr_col;
      vcol[cb] = vrow * ROWB + (((col >> 3) ^ stream::key_v(vrow)) << 4) + (col & 7) * 2;
    }
  }

  f32x16 oacc[HD / 32];
#pragma unroll
  for (int cb = 0; cb < HD / 32; ++cb) oacc[cb] = f32x16{};
  float m_run = NEG_BIG, l_run = 0.f;
  f32x16 sacc[2];   // scores of the group's newest tile, then its probabilities
  bf16x8 pb[4];     // probabilities of the previous tile, one fragment per 16-key step
#pragma unroll
  for (int kb = 0; kb < 2; ++kb) sacc[kb] = f32x16{};
#pragma unroll
  for (int st = 0; st < 4; ++st) pb[st] = bf16x8{};

  // MFMA phase k: O^T += V^T P^T of tile k - 1, then the scores of tile k.
  auto mma_phase = [&](int k) {
    if (k >= 1 && k - 1 < nj) {
      // V^T fragments in two halves of 32 keys (16 transpose reads each), each waited for just
      // before its MFMAs.
      const uint32_t vs = lds_addr(gbase + 2 * TILE_BYTES + ((k - 1) & 1) * TILE_BYTES);
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        s16x4 vbuf[2][2 * (HD / 32)];
        if (h == 0) {
          read_v_step<ROWB, 0>(vs, vcol, vbuf[0]);
          read_v_step<ROWB, 16>(vs, vcol, vbuf[1]);
        } else {
          read_v_step<ROWB, 32>(vs, vcol, vbuf[0]);
          read_v_step<ROWB, 48>(vs, vcol, vbuf[1]);
        }
        lds_wait(vbuf[0]);
        lds_wait(vbuf[1]);
#pragma unroll
        for (int s2 = 0; s2 < 2; ++s2)
#pragma unroll
          for (int cb = 0; cb < HD / 32; ++cb) {
            const s16x4 vv[2] = {vbuf[s2][2 * cb], vbuf[s2][2 * cb + 1]};
            mfma_k16(oacc[cb], __builtin_bit_cast(bf16x8, vv), pb[2 * h + s2]);
          }
      }
    }
    if (k < nj) {
      const unsigned char* sk = gbase + (k & 1) * TILE_BYTES;
      // The two 32-key score chains interleaved (K step outer): consecutive MFMAs are independent.
      sacc[0] = f32x16{};
      sacc[1] = f32x16{};
#pragma unroll
      for (int ks = 0; ks < HD / 16; ++ks)
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
          const int row = kb * 32 + (lane & 31);
          const int chunk = ks * 2 + g2;
          bf16x8 kf = __builtin_bit_cast(
              bf16x8, *(const u32x4*)(sk + row * ROWB + ((chunk ^ stream::key_k(row)) << 4)));
          mfma_k16(sacc[kb], kf, qf[ks]);
        }
    }
  };
  // Softmax phase k (k >= 0). Every wave of the group finished MFMA phase k (the barrier before
  // this phase), so the slots of K tile k and V tile k - 1 are free: refill them with K tile
  // k + 2 and V tile k + 1; then the probabilities of tile k.
  auto softmax_phase = [&](int k) {
    issue(k + 2, KTag{});
    issue(k + 1, VTag{});
    if (k < nj) {
      const int t = t_begin + grp + 2 * k;
      const bool vis = t < tv;
      const int key0 = (vis ? t : t - tv) * KT;
      if (!vis || key0 + KT > a.Nv) {  // partial visual tile or text tile: mask
        const int last = (vis ? a.Nv - 1 : min(my_text_last, text_lim - 1)) - key0;
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int i = 0; i < 16; ++i)
            sacc[kb][i] = kb * 32 + acc_row(lane, i) > last ? -INFINITY : sacc[kb][i];
      }
      online_softmax(sacc, a.scale_log2, m_run, l_run, oacc);
      // K step st = (kb, s2) of the P V product takes slots s2 * 8 .. + 7 of key block kb.
      float lsum[2] = {0.f, 0.f};
#pragma unroll
      for (int st = 0; st < 4; ++st) {
        const int kb = st >> 1, s2 = st & 1;
#pragma unroll
        for (int e = 0; e < 8; ++e) pb[st][e] = (bf16)sacc[kb][s2 * 8 + e];
        lsum[s2] = add_probs(pb[st], lsum[s2]);
      }
      l_run += lsum[0] + lsum[1];
    }
  };
  // Period q: the first group runs MFMA phase q and then softmax phase q, the second group
  // softmax phase q - 1 and then MFMA phase q. Before each half every wave has at most its
  // latest refill (two tiles' loads) in flight, so the tiles of an MFMA phase have landed, and
  // its LDS reads have returned.
  // One loop per group, each with two barriers per period, so each wave's program is a plain
  // sequence of its own phases.
  const int nq = nA + 1;
  if (grp == 0) {
    for (int q = 0; q < nq; ++q) {
      pipe_sync<waitcnt_imm(2 * LD, 0)>();
      mma_phase(q);
      pipe_sync<waitcnt_imm(2 * LD, 0)>();
      softmax_phase(q);
    }
  } else {
    for (int q = 0; q < nq; ++q) {
      pipe_sync<waitcnt_imm(2 * LD, 0)>();
      if (q >= 1) softmax_phase(q - 1);
      pipe_sync<waitcnt_imm(2 * LD, 0)>();
      mma_phase(q);
    }
  }
  // The last refills (past the end: zeros) land before the rings are reused for the merge.
  pipe_sync<waitcnt_imm(0, 0)>();

  const float l_tot = l_run + shfl_xor(l_run, 32);
  float* red_o = (float*)smem;                 // [NRW][32 rows][MPITCH]: the second group's O^T
  float* red_ml = red_o + NRW * 32 * MPITCH;   // [NRW][32 rows][2]
  const int rrow = lane & 31;
  if (grp == 1) {
    float* o = red_o + (rw * 32 + rrow) * MPITCH;
#pragma unroll
    for (int cb = 0; cb < HD / 32; ++cb)
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        const int c = cb * 32 + q4 * 8 + g2 * 4;
        *(f32x4*)(o + c) = f32x4{oacc[cb][q4 * 4], oacc[cb][q4 * 4 + 1], oacc[cb][q4 * 4 + 2],
                                 oacc[cb][q4 * 4 + 3]};
      }
    if (g2 == 0) {
      red_ml[(rw * 32 + rrow) * 2] = m_run;
      red_ml[(rw * 32 + rrow) * 2 + 1] = l_tot;
    }
  }
  __syncthreads();
  if (grp == 1 || !row_ok) return;  // no barrier follows
  const float m_o = red_ml[(rw * 32 + rrow) * 2], l_o = red_ml[(rw * 32 + rrow) * 2 + 1];
  const float mx = fmaxf(m_run, m_o);
  const float sa = __builtin_amdgcn_exp2f(m_run - mx), sb = __builtin_amdgcn_exp2f(m_o - mx);
  const float lt = l_tot * sa + l_o * sb;
  const float* o2 = red_o + (rw * 32 + rrow) * MPITCH;
  const int64_t orow = ((int64_t)b * a.Nq + my_i) * a.Hq + my_h;
  const int64_t rows_total = (int64_t)a.B * a.Nq * a.Hq;
  const float inv = lt > 0.f ? 1.f / lt : 0.f;
#pragma unroll
  for (int cb = 0; cb < HD / 32; ++cb)
#pragma unroll
    for (int q4 = 0; q4 < 4; ++q4) {
      const int c = cb * 32 + q4 * 8 + g2 * 4;
      const f32x4 ob = *(const f32x4*)(o2 + c);
      float y[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) y[u] = oacc[cb][q4 * 4 + u] * sa + ob[u] * sb;
      if (a.splits == 1)
        store4<bf16>((bf16*)a.O + orow * HD + c, y[0] * inv, y[1] * inv, y[2] * inv, y[3] * inv);
      else
        *(f32x4*)(a.Opart + ((int64_t)split * rows_total + orow) * HD + c) =
            f32x4{y[0], y[1], y[2], y[3]};
    }
  if (a.splits > 1 && g2 == 0) {
    float* ml = a.MLpart + ((int64_t)split * rows_total + orow) * 2;
    ml[0] = mx;
    ml[1] = lt;
  }
}

// ------------------------------------------------------------------ key-split prefill (bf16)
//
// For few query rows per (batch, kv-head) (LLaVA: 64) one block of four waves takes 32 rows
// and every wave streams a quarter of the 32-key tiles through its own two LDS stages, so all
// four SIMDs of the CU work and no barrier is needed until the waves merge their partial
// (max, sum, O) through LDS. At most two blocks read a tile, one right after the other, and
// the tiles are loaded non-temporally (LLaVA-7B: about 3% faster than the default policy).

namespace ksplit {
constexpr int HD = 128;
constexpr int KT = 32;                      // keys per tile
constexpr int NWAVE = 4;                    // key groups per block
constexpr int ROWB = HD * 2;
constexpr int TILE_BYTES = KT * ROWB;       // 8 KiB per tensor
constexpr int STAGE_BYTES = 2 * TILE_BYTES;
constexpr int NS = 2;
constexpr int WAVE_BYTES = NS * STAGE_BYTES;
constexpr int LDS_BYTES = NWAVE * WAVE_BYTES;  // 128 KiB; the merge reuses it
constexpr int INS = 2 * KT / 4;             // 1 KiB load instructions per tile
constexpr int MPITCH = HD + 4;              // merge rows padded by 16 B: rows fall on distinct banks
static_assert(NWAVE * 32 * (MPITCH + 2) * 4 <= LDS_BYTES, "merge buffer must fit");
}  // namespace ksplit

__global__ __launch_bounds__(ksplit::NWAVE * 64) void k_attn_ksplit(AttnArgs a, int row_blocks) {
  using namespace ksplit;
  extern __shared__ __align__(16) unsigned char smem[];

  const int lane = threadIdx.x & 63, wave = wave_index(), g2 = lane >> 5;
  const int G = a.Hq / a.Hkv, R = a.Nq * G, n_bg = a.B * a.Hkv;
  const BlockWork wk = block_work(n_bg, row_blocks, a.splits);
  const int rb = wk.rb, bg = wk.bg, split = wk.split;
  const int b = uni(bg / a.Hkv), g = bg - b * a.Hkv;
  const int row0 = rb * 32;
  const int my_row = row0 + (lane & 31);
  const bool row_ok = my_row < R;
  const int my_i = row_ok ? my_row / G : 0;
  const int my_h = g * G + (row_ok ? my_row - my_i * G : 0);
  const int i_max = uni((min(row0 + 32, R) - 1) / G);
  const int text_lim = min(a.Nkt, a.q_pos0 + i_max + 1);
  const int my_text_last = a.q_pos0 + my_i;
  const int tv = uni((a.Nv + KT - 1) / KT), ntiles = uni(tv + (text_lim + KT - 1) / KT);
  const int t_begin = split * a.tiles_per_split;
  const int t_end = min(ntiles, t_begin + a.tiles_per_split);

  const bf16* kvb = (const bf16*)a.Kv + (int64_t)bg * a.Nv * HD;
  const bf16* vvb = (const bf16*)a.Vv + (int64_t)bg * a.Nv * HD;
  const bf16* ktb = (const bf16*)a.Kt + (int64_t)bg * a.Nkt * HD;
  const bf16* vtb = (const bf16*)a.Vt + (int64_t)bg * a.Nkt * HD;
  const int64_t vis_bytes = (int64_t)a.Nv * ROWB, txt_bytes = (int64_t)text_lim * ROWB;

  bf16x8 qf[HD / 16];
  {
    const bf16* qrow = (const bf16*)a.Q + (((int64_t)b * a.Nq + my_i) * a.Hq + my_h) * HD;
#pragma unroll
    for (int ks = 0; ks < HD / 16; ++ks)
      qf[ks] = row_ok ? __builtin_bit_cast(bf16x8, ld16(qrow + ks * 16 + g2 * 8)) : bf16x8{};
  }

  unsigned char* mine = smem + wave * WAVE_BYTES;  // this wave's two stages
  const int r4 = lane >> 4, pc = lane & 15;
  auto issue = [&](int t, int stage) {
    const bool vis = t < tv;
    const int key0 = (vis ? t : t - tv) * KT;
    unsigned char* sk = mine + stage * STAGE_BYTES;
    unsigned char* sv = sk + TILE_BYTES;
    const __amdgpu_buffer_rsrc_t rk = buffer_rsrc(vis ? kvb : ktb, vis ? vis_bytes : txt_bytes);
    const __amdgpu_buffer_rsrc_t rv = buffer_rsrc(vis ? vvb : vtb, vis ? vis_bytes : txt_bytes);
#pragma unroll
    for (int blk = 0; blk < KT / 4; ++blk) {
      const int row = blk * 4 + r4;
      const int soff = (key0 + blk * 4) * ROWB;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rk, (lds_void*)(sk + blk * 1024), 16,
                                               r4 * ROWB + ((pc ^ stream::key_k(row)) << 4), soff,
                                               0, stream::CPOL_NT);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rv, (lds_void*)(sv + blk * 1024), 16,
                                               r4 * ROWB + ((pc ^ stream::key_v(row)) << 4), soff,
                                               0, stream::CPOL_NT);
    }
  };

  f32x16 oacc[HD / 32];
#pragma unroll
  for (int cb = 0; cb < HD / 32; ++cb) oacc[cb] = f32x16{};
  float m_run = NEG_BIG, l_run = 0.f;

  const int l16 = lane & 15, grp = lane >> 4;
  const int tr_row = l16 >> 2;
  const int tr_col = 16 * (grp & 1) + 4 * (l16 & 3);
  uint32_t vcol[4];  // as in k_attn_stream
  {
    const int vrow = 4 * (grp >> 1) + tr_row;
#pragma unroll
    for (int cb = 0; cb < 4; ++cb) {
      const int col = 32 * cb + tr_col;
      vcol[cb] = vrow * ROWB + (((col >> 3) ^ stream::key_v(vrow)) << 4) + (col & 7) * 2;
    }
  }

  // My tiles: t_begin + wave, + NWAVE, ...  Only this wave reads its stages: waits only.
  int t = t_begin + wave;
  if (t < t_end) issue(t, 0);
  if (t + NWAVE < t_end) issue(t + NWAVE, 1);
  int stage = 0;
  for (; t < t_end; t += NWAVE) {
    if (t + NWAVE < t_end) __builtin_amdgcn_s_waitcnt(waitcnt_imm(INS, 0));
    else __builtin_amdgcn_s_waitcnt(waitcnt_imm(0, 0));
    asm volatile("" ::: "memory");
    const unsigned char* sk = mine + stage * STAGE_BYTES;
    const unsigned char* sv = sk + TILE_BYTES;
    const bool vis = t < tv;
    const int key0 = (vis ? t : t - tv) * KT;

    // V^T fragments of both K steps, read now so that they land during the scores and softmax
    // (one wave per SIMD: registers are plentiful). Slot e of lane half g2 in K step s2 is key
    // 16*s2 + (e/4)*8 + 4*g2 + e%4 in both operands; the two transpose loads return slots 0..3
    // and 4..7 of V^T for column 32*cb + lane % 32.
    s16x4 vr[2][2 * (HD / 32)];
    const uint32_t vs = lds_addr(sv);
    read_v_step<ROWB, 0>(vs, vcol, vr[0]);
    read_v_step<ROWB, 16>(vs, vcol, vr[1]);

    f32x16 sacc[1] = {f32x16{}};
    {
      const int row = lane & 31;
#pragma unroll
      for (int ks = 0; ks < HD / 16; ++ks) {
        const int chunk = ks * 2 + g2;
        bf16x8 kf = __builtin_bit_cast(
            bf16x8, *(const u32x4*)(sk + row * ROWB + ((chunk ^ stream::key_k(row)) << 4)));
        mfma_k16(sacc[0], kf, qf[ks]);
      }
    }
    if (!vis || key0 + KT > a.Nv) {  // partial visual tile or text tile: mask (as above)
      const int last = (vis ? a.Nv - 1 : min(my_text_last, text_lim - 1)) - key0;
#pragma unroll
      for (int i = 0; i < 16; ++i) sacc[0][i] = acc_row(lane, i) > last ? -INFINITY : sacc[0][i];
    }
    online_softmax(sacc, a.scale_log2, m_run, l_run, oacc);
    lds_wait(vr[0]);
    lds_wait(vr[1]);
    float lsum[2] = {0.f, 0.f};
#pragma unroll
    for (int s2 = 0; s2 < 2; ++s2) {
      bf16x8 pf;
#pragma unroll
      for (int e = 0; e < 8; ++e) pf[e] = (bf16)sacc[0][s2 * 8 + e];
      lsum[s2] = add_probs(pf, lsum[s2]);
#pragma unroll
      for (int cb = 0; cb < HD / 32; ++cb) {
        const s16x4 vv[2] = {vr[s2][2 * cb], vr[s2][2 * cb + 1]};
        mfma_k16(oacc[cb], __builtin_bit_cast(bf16x8, vv), pf);
      }
    }
    l_run += lsum[0] + lsum[1];
    // This stage is consumed (lgkmcnt drained) before it is refilled with tile t + 2*NWAVE.
    __builtin_amdgcn_s_waitcnt(waitcnt_imm(63, 0));
    asm volatile("" ::: "memory");
    if (t + 2 * NWAVE < t_end) issue(t + 2 * NWAVE, stage);
    stage ^= 1;
  }
  const float l_mine = l_run + shfl_xor(l_run, 32);

  // Merge the four key groups: every wave publishes (m, l, O^T) and wave w finishes columns
  // 32w .. 32w + 31 of the block's 32 rows.
  __syncthreads();
  float* red_o = (float*)smem;                        // [NWAVE][32 rows][MPITCH]
  float* red_ml = red_o + NWAVE * 32 * MPITCH;        // [NWAVE][32 rows][2]
  {
    const int rrow = lane & 31;
    float* o = red_o + (wave * 32 + rrow) * MPITCH;
#pragma unroll
    for (int cb = 0; cb < HD / 32; ++cb)
#pragma unroll
      for (int q4 = 0; q4 < 4; ++q4) {
        const int c = cb * 32 + q4 * 8 + g2 * 4;
        *(f32x4*)(o + c) = f32x4{oacc[cb][q4 * 4], oacc[cb][q4 * 4 + 1], oacc[cb][q4 * 4 + 2],
                                 oacc[cb][q4 * 4 + 3]};
      }
    if (g2 == 0) {
      red_ml[(wave * 32 + rrow) * 2] = m_run;
      red_ml[(wave * 32 + rrow) * 2 + 1] = l_mine;
    }
  }
  __syncthreads();
  const int rrow = lane & 31;
  float mx = NEG_BIG;
#pragma unroll
  for (int w = 0; w < NWAVE; ++w) mx = fmaxf(mx, red_ml[(w * 32 + rrow) * 2]);
  float lt = 0.f, sc[NWAVE];
#pragma unroll
  for (int w = 0; w < NWAVE; ++w) {
    sc[w] = __builtin_amdgcn_exp2f(red_ml[(w * 32 + rrow) * 2] - mx);
    lt += red_ml[(w * 32 + rrow) * 2 + 1] * sc[w];
  }
  if (!row_ok) return;
  const int64_t orow = ((int64_t)b * a.Nq + my_i) * a.Hq + my_h;
  const int cbase = wave * 32 + g2 * 16;  // this lane's 16 columns
  float out[16];
#pragma unroll
  for (int e = 0; e < 16; ++e) out[e] = 0.f;
#pragma unroll
  for (int w = 0; w < NWAVE; ++w) {
    const float* o = red_o + (w * 32 + rrow) * MPITCH + cbase;
#pragma unroll
    for (int e4 = 0; e4 < 4; ++e4) {
      const f32x4 v = *(const f32x4*)(o + e4 * 4);
#pragma unroll
      for (int u = 0; u < 4; ++u) out[e4 * 4 + u] += v[u] * sc[w];
    }
  }
  if (a.splits == 1) {
    const float inv = lt > 0.f ? 1.f / lt : 0.f;
    bf16* op = (bf16*)a.O + orow * HD + cbase;
#pragma unroll
    for (int e4 = 0; e4 < 4; ++e4)
      store4<bf16>(op + e4 * 4, out[e4 * 4] * inv, out[e4 * 4 + 1] * inv, out[e4 * 4 + 2] * inv,
                   out[e4 * 4 + 3] * inv);
  } else {
    const int64_t rows_total = (int64_t)a.B * a.Nq * a.Hq;
    float* op = a.Opart + ((int64_t)split * rows_total + orow) * HD + cbase;
#pragma unroll
    for (int e4 = 0; e4 < 4; ++e4)
      *(f32x4*)(op + e4 * 4) = f32x4{out[e4 * 4], out[e4 * 4 + 1], out[e4 * 4 + 2], out[e4 * 4 + 3]};
    if (wave == 0 && g2 == 0) {
      float* ml = a.MLpart + ((int64_t)split * rows_total + orow) * 2;
      ml[0] = mx;
      ml[1] = lt;
    }
  }
}

// ------------------------------------------------------------------ decode

template <typename T, int HD, int MAXG>
__global__ __launch_bounds__(256) void k_attn_decode(AttnArgs a) {
  constexpr int NW = 4;
  constexpr int LPK = HD / 8;      // lanes per key row (8 elements each)
  constexpr int KPW = WAVE / LPK;  // keys per wave step
  constexpr int U = 4;             // key steps in flight per lane
  __shared__ float red_m[NW][MAXG], red_l[NW][MAXG];
  __shared__ float red_o[NW][MAXG][HD];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int sub = lane % LPK, grp = lane / LPK;
  const int G = a.Hq / a.Hkv;
  const int bg = blockIdx.x, b = bg / a.Hkv, g = bg - b * a.Hkv;
  const int split = blockIdx.y;
  const int nk = a.Nv + a.q_pos0 + 1;  // the single query sees every visual key and text 0..q_pos0
  const int k_begin = split * a.keys_per_split;
  const int k_end = min(nk, k_begin + a.keys_per_split);

  const T* Kvb = (const T*)a.Kv + (int64_t)bg * a.Nv * HD + sub * 8;
  const T* Vvb = (const T*)a.Vv + (int64_t)bg * a.Nv * HD + sub * 8;
  const T* Ktb = (const T*)a.Kt + (int64_t)bg * a.Nkt * HD + sub * 8;
  const T* Vtb = (const T*)a.Vt + (int64_t)bg * a.Nkt * HD + sub * 8;

  float q[MAXG][8], o[MAXG][8], m[MAXG], l[MAXG];
#pragma unroll
  for (int h = 0; h < MAXG; ++h) {
    m[h] = NEG_BIG;
    l[h] = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) o[h][e] = 0.f;
    if (h < G) {
      load_row8_f32<T>((const T*)a.Q + ((int64_t)b * a.Hq + g * G + h) * HD + sub * 8, q[h]);
#pragma unroll
      for (int e = 0; e < 8; ++e) q[h][e] *= a.scale_log2;
    }
  }

  const int stride = NW * KPW;
  for (int j0 = k_begin + wave * KPW + grp; j0 < k_end; j0 += stride * U) {
    // Rows stay in their storage type until used (bf16: 4 registers per 8 elements): converted on
    // load they took 64 registers, leaving four waves per SIMD instead of five (about 2% on the
    // B 64 decode shape, bit-identical). The cache rows are read exactly once, so they are loaded
    // non-temporally and do not displace reusable lines from the L2 and the MALL (B 64 decode:
    // 5.70-5.91 -> 6.37 TB/s).
    u32x4 kr[U][sizeof(T) / 2], vr[U][sizeof(T) / 2];
    bool ok[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int j = j0 + u * stride;
      ok[u] = j < k_end;
      const T* kp = j < a.Nv ? Kvb + (int64_t)j * HD : Ktb + (int64_t)(j - a.Nv) * HD;
      const T* vp = j < a.Nv ? Vvb + (int64_t)j * HD : Vtb + (int64_t)(j - a.Nv) * HD;
#pragma unroll
      for (int q2 = 0; q2 < (int)(sizeof(T) / 2); ++q2) {
        kr[u][q2] = ok[u] ? ld16_stream(kp + q2 * (8 / (sizeof(T) / 2))) : u32x4{};
        vr[u][q2] = ok[u] ? ld16_stream(vp + q2 * (8 / (sizeof(T) / 2))) : u32x4{};
      }
    }
    auto unpack = [&](const u32x4 (&r)[sizeof(T) / 2], float (&x)[8]) {
      if constexpr (sizeof(T) == 2) {
        const bf16x8 v = __builtin_bit_cast(bf16x8, r[0]);
#pragma unroll
        for (int e = 0; e < 8; ++e) x[e] = (float)v[e];
      } else {
        // Whole vectors are reinterpreted: a bit_cast of one vector element read the wrong bytes
        // (the compiler narrowed the 16-byte loads to their first dword).
        const f32x4 v0 = __builtin_bit_cast(f32x4, r[0]), v1 = __builtin_bit_cast(f32x4, r[1]);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          x[e] = v0[e];
          x[4 + e] = v1[e];
        }
      }
    };

#pragma unroll
    for (int h = 0; h < MAXG; ++h) {
      if (h >= G) break;
      float s[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        float acc = 0.f;
        float kx[8];
        unpack(kr[u], kx);
#pragma unroll
        for (int e = 0; e < 8; ++e) acc = fmaf(q[h][e], kx[e], acc);
#pragma unroll
        for (int w = 1; w < LPK; w <<= 1) acc += shfl_xor(acc, w);
        s[u] = ok[u] ? acc : -INFINITY;
      }
      float mx = m[h];
#pragma unroll
      for (int u = 0; u < U; ++u) mx = fmaxf(mx, s[u]);
      const float alpha = exp2f(m[h] - mx);
      m[h] = mx;
      float ps = 0.f;
#pragma unroll
      for (int e = 0; e < 8; ++e) o[h][e] *= alpha;
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const float p = exp2f(s[u] - mx);
        ps += p;
        float vx[8];
        unpack(vr[u], vx);
#pragma unroll
        for (int e = 0; e < 8; ++e) o[h][e] = fmaf(p, vx[e], o[h][e]);
      }
      l[h] = l[h] * alpha + ps;
    }
  }

  // Merge the key groups of the wave (lanes differing in the bits above LPK).
#pragma unroll
  for (int w = LPK; w < WAVE; w <<= 1) {
#pragma unroll
    for (int h = 0; h < MAXG; ++h) {
      if (h >= G) break;
      const float mo = shfl_xor(m[h], w), lo = shfl_xor(l[h], w);
      const float mx = fmaxf(m[h], mo);
      const float sa = exp2f(m[h] - mx), sb = exp2f(mo - mx);
      l[h] = l[h] * sa + lo * sb;
#pragma unroll
      for (int e = 0; e < 8; ++e) o[h][e] = o[h][e] * sa + shfl_xor(o[h][e], w) * sb;
      m[h] = mx;
    }
  }
  if (grp == 0) {
#pragma unroll
    for (int h = 0; h < MAXG; ++h) {
      if (h >= G) break;
#pragma unroll
      for (int e = 0; e < 8; ++e) red_o[wave][h][sub * 8 + e] = o[h][e];
      if (sub == 0) {
        red_m[wave][h] = m[h];
        red_l[wave][h] = l[h];
      }
    }
  }
  __syncthreads();
  // Merge the waves: thread t handles (head h, channel c).
  for (int t = tid; t < G * HD; t += NW * WAVE) {
    const int h = t / HD, c = t - h * HD;
    float mx = NEG_BIG;
#pragma unroll
    for (int w = 0; w < NW; ++w) mx = fmaxf(mx, red_m[w][h]);
    float lt = 0.f, ot = 0.f;
#pragma unroll
    for (int w = 0; w < NW; ++w) {
      const float sc = exp2f(red_m[w][h] - mx);
      lt += red_l[w][h] * sc;
      ot += red_o[w][h][c] * sc;
    }
    const int64_t orow = (int64_t)b * a.Hq + g * G + h;
    if (a.splits == 1) {
      ((T*)a.O)[orow * HD + c] = from_f32<T>(lt > 0.f ? ot / lt : 0.f);
    } else {
      const int64_t rows_total = (int64_t)a.B * a.Hq;
      a.Opart[((int64_t)split * rows_total + orow) * HD + c] = ot;
      if (c == 0) {
        float* ml = a.MLpart + ((int64_t)split * rows_total + orow) * 2;
        ml[0] = mx;
        ml[1] = lt;
      }
    }
  }
}

// ------------------------------------------------------------------ combine

template <typename T, int HD>
__global__ __launch_bounds__(256) void k_attn_combine(const float* __restrict__ Opart,
                                                      const float* __restrict__ MLpart,
                                                      T* __restrict__ O, int64_t rows, int splits) {
  const int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  constexpr int CPR = HD / 4;
  if (t >= rows * CPR) return;
  const int64_t row = t / CPR;
  const int c = (int)(t - row * CPR) * 4;
  // Unrolled so that several splits' loads are in flight at once: the partials were written by
  // blocks on every XCD and come from beyond this XCD's L2.
  float mx = NEG_BIG;
#pragma unroll 8
  for (int s = 0; s < splits; ++s) mx = fmaxf(mx, MLpart[((int64_t)s * rows + row) * 2]);
  float lt = 0.f;
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll 8
  for (int s = 0; s < splits; ++s) {
    const float* ml = MLpart + ((int64_t)s * rows + row) * 2;
    const float sc = exp2f(ml[0] - mx);
    lt += ml[1] * sc;
    acc += *(const f32x4*)(Opart + ((int64_t)s * rows + row) * HD + c) * sc;
  }
  const float inv = lt > 0.f ? 1.f / lt : 0.f;
  store4<T>(O + row * HD + c, acc[0] * inv, acc[1] * inv, acc[2] * inv, acc[3] * inv);
}

// ------------------------------------------------------------------ host side

static inline int64_t cdiv64(int64_t x, int64_t y) { return (x + y - 1) / y; }

AttnPlan plan_attention(int B, int Hq, int Hkv, int hd, int Nv, int Nq, int Nkt, int q_pos0,
                        int dtype, size_t ws_bytes) {
  AttnPlan p{};
  const int G = Hq / Hkv;
  const int64_t rows_total = (int64_t)B * Nq * Hq;
  const int64_t per_split = rows_total * (int64_t)(hd + 2) * 4;
  const int max_keys = Nv + q_pos0 + Nq;  // keys seen by the last query
  const int n_bg = B * Hkv;
  p.decode = (Nq == 1 && G <= 8);
  p.stream = !p.decode && dtype == 1 && hd == 128;
  int64_t units, tiles;
  int64_t min_blocks = 512;
  if (p.decode) {
    p.nw = 4;
    units = n_bg;
    tiles = cdiv64(max_keys, 64);
  } else if (p.stream) {
    const int R = Nq * G;
    p.ksplit = R <= 64;
    if (p.ksplit) {
      // Few rows: blocks of 32 rows whose four waves split the key tiles (32 keys each).
      p.nw = 4;
      p.row_blocks = (int)cdiv64(R, 32);
      tiles = cdiv64(Nv, 32) + cdiv64(std::min(Nkt, q_pos0 + Nq), 32);
    } else {
      // Many rows share each K/V tile (64-key tiles): up to 96 rows the two-wave streaming
      // kernel, above that the ping-pong kernel (blocks of 128 rows).
      p.pp = R > 96;
      p.nw = p.pp ? 4 : 2;  // 32-row waves per row block (the ping-pong kernel runs two such groups)
      p.row_blocks = (int)cdiv64(R, 32 * p.nw);
      tiles = cdiv64(Nv, 64) + cdiv64(std::min(Nkt, q_pos0 + Nq), 64);
    }
    units = (int64_t)n_bg * p.row_blocks;
    min_blocks = 256;
  } else {
    const int R = Nq * G;
    p.nw = R <= 32 ? 1 : (R <= 64 ? 2 : 4);
    p.row_blocks = (int)cdiv64(R, 32 * p.nw);
    units = (int64_t)n_bg * p.row_blocks;
    tiles = cdiv64(max_keys, 64);
  }
  // Split keys only when the blocks do not fill the chip; keep at least two tiles per split.
  int64_t want = units >= min_blocks ? 1 : cdiv64(min_blocks, units);
  want = std::min<int64_t>(want, std::max<int64_t>(1, tiles / 2));
  want = std::max<int64_t>(1, std::min<int64_t>(want, 64));
  const int64_t fit = per_split > 0 ? (int64_t)(ws_bytes / (size_t)per_split) : 0;
  // Both streaming kernels hold one block per CU (LDS), so they run in rounds of 256 blocks.
  static_assert(stream::blocks_per_cu<2>() == 1, "two-wave streaming blocks: one per CU");
  const int64_t slots = 256;
  if (p.stream && !p.ksplit && units < 256) {
    // Take the split count with the fewest tile steps over all rounds,
    // rounds(units * S) * ceil(tiles / S), preferring fewer splits on ties. Keys are split only
    // while some CU would have no block: with four-wave blocks two to a CU, LLaVA-NeXT's 256
    // streams (128 rows per kv-head) ran 84 us per layer unsplit against 88 us for two
    // half-range blocks per CU and their merge.
    int64_t best = 1, best_cost = tiles;
    const int64_t smax = std::min<int64_t>(64, std::max<int64_t>(1, tiles / 2));
    for (int64_t sp = 2; sp <= smax && sp <= fit; ++sp) {
      const int64_t cost = cdiv64(units * sp, slots) * cdiv64(tiles, sp);
      if (cost < best_cost) {
        best = sp;
        best_cost = cost;
      }
    }
    want = best;
  } else if (want > 1 && per_split > 0) {
    want = std::min<int64_t>(want, fit);
    if (want < 2) want = 1;
  }
  const int64_t tiles_per_split = cdiv64(tiles, want);
  p.tiles_per_split = (int)tiles_per_split;
  p.keys_per_split = (int)(tiles_per_split * 64);
  p.splits = (int)cdiv64(tiles, tiles_per_split);  // drop empty trailing splits
  p.ws_needed = p.splits > 1 ? (size_t)(p.splits * per_split) : 0;
  return p;
}

size_t attention_workspace(int B, int Hq, int Hkv, int hd, int Nv, int Nq, int Nkt) {
  // The largest need over both dtypes and every valid q_pos0 (more keys never mean fewer splits).
  const AttnPlan p0 = plan_attention(B, Hq, Hkv, hd, Nv, Nq, Nkt, Nkt - Nq, 0, (size_t)-1);
  const AttnPlan p1 = plan_attention(B, Hq, Hkv, hd, Nv, Nq, Nkt, Nkt - Nq, 1, (size_t)-1);
  return std::max(p0.ws_needed, p1.ws_needed);
}

template <typename T, int HD>
static hipError_t attn_launch_t(const AttnArgs& a, const AttnPlan& p, hipStream_t s,
                                const LaunchEvents& ev) {
  record(ev.attn[0], s);
  if (p.decode) {
    dim3 grid(a.B * a.Hkv, p.splits);
    const int G = a.Hq / a.Hkv;
    if (G == 1)
      k_attn_decode<T, HD, 1><<<grid, dim3(256), 0, s>>>(a);
    else if (G == 2)
      k_attn_decode<T, HD, 2><<<grid, dim3(256), 0, s>>>(a);
    else if (G <= 4)
      k_attn_decode<T, HD, 4><<<grid, dim3(256), 0, s>>>(a);
    else
      k_attn_decode<T, HD, 8><<<grid, dim3(256), 0, s>>>(a);
  } else if (p.stream) {
    if constexpr (sizeof(T) == 2 && HD == 128) {
      using stream::CPOL_DEFAULT;
      using stream::CPOL_NT;
      static bool once = [] {
        (void)hipFuncSetAttribute((const void*)k_attn_stream<2, CPOL_DEFAULT>,
                                  hipFuncAttributeMaxDynamicSharedMemorySize, stream::lds_bytes<2>());
        (void)hipFuncSetAttribute((const void*)k_attn_pp<CPOL_DEFAULT>,
                                  hipFuncAttributeMaxDynamicSharedMemorySize, pp::LDS_BYTES);
        (void)hipFuncSetAttribute((const void*)k_attn_pp<CPOL_NT>,
                                  hipFuncAttributeMaxDynamicSharedMemorySize, pp::LDS_BYTES);
        return true;
      }();
      (void)once;
      dim3 grid(a.B * a.Hkv * p.row_blocks, p.splits);
      if (p.ksplit) {
        static bool once_k = [] {
          (void)hipFuncSetAttribute((const void*)k_attn_ksplit,
                                    hipFuncAttributeMaxDynamicSharedMemorySize, ksplit::LDS_BYTES);
          return true;
        }();
        (void)once_k;
        k_attn_ksplit<<<grid, dim3(ksplit::NWAVE * 64), ksplit::LDS_BYTES, s>>>(a, p.row_blocks);
      } else if (p.pp) {
        if (p.row_blocks == 1)  // each tile has one reader
          k_attn_pp<CPOL_NT><<<grid, dim3(pp::NWAVE * 64), pp::LDS_BYTES, s>>>(a, p.row_blocks);
        else
          k_attn_pp<CPOL_DEFAULT><<<grid, dim3(pp::NWAVE * 64), pp::LDS_BYTES, s>>>(a, p.row_blocks);
      } else {
        k_attn_stream<2, CPOL_DEFAULT><<<grid, dim3(128), stream::lds_bytes<2>(), s>>>(a, p.row_blocks);
      }
    } else {
      return hipErrorInvalidValue;  // the planner only picks this kernel for bf16, hd 128
    }
  } else {
    // bf16 hd-128 prefill always takes the streaming kernels, so no such instance is built.
    if constexpr (sizeof(T) == 2 && HD == 128) {
      return hipErrorInvalidValue;
    } else {
      dim3 grid(p.row_blocks, a.B * a.Hkv, p.splits);
      if (p.nw == 1)
        k_attn_prefill<T, HD, 1><<<grid, dim3(64), AttnCfg<T, HD, 1>::LDS_BYTES, s>>>(a);
      else if (p.nw == 2)
        k_attn_prefill<T, HD, 2><<<grid, dim3(128), AttnCfg<T, HD, 2>::LDS_BYTES, s>>>(a);
      else
        k_attn_prefill<T, HD, 4><<<grid, dim3(256), AttnCfg<T, HD, 4>::LDS_BYTES, s>>>(a);
    }
  }
  record(ev.attn[1], s);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || p.splits == 1) return e;
  const int64_t rows = (int64_t)a.B * a.Nq * a.Hq;
  const int64_t threads = rows * (HD / 4);
  k_attn_combine<T, HD><<<dim3((unsigned)cdiv64(threads, 256)), dim3(256), 0, s>>>((const float*)a.Opart, (const float*)a.MLpart, (T*)a.O, rows, p.splits);
  return hipGetLastError();
}

// ------------------------------------------------------------------ static scratch
//
// Key-split partials of dv_text_visual_attention_noalloc, for callers that cannot allocate. Each
// GPU holds its own copy of this array for the life of the process. In host code `scratch` names
// a host-side stand-in, not device memory: kernels get the device address that
// hipGetSymbolAddress returns for the current device, looked up once per device.

static __device__ __align__(256) unsigned char scratch[DV_ATTENTION_SCRATCH_BYTES];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};
}  // namespace

size_t attention_scratch_bytes() { return DV_ATTENTION_SCRATCH_BYTES; }

hipError_t attention_scratch(void** ptr) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (!p) return hipErrorInvalidSymbol;
    g_scratch_ptr[dev] = p;
  }
  *ptr = g_scratch_ptr[dev];
  return hipSuccess;
}

hipError_t launch_attention(const AttnArgs& a, const AttnPlan& p, int dtype, hipStream_t s,
                            const LaunchEvents& ev) {
  if (dtype == 1) {
    if (a.hd == 128) return attn_launch_t<bf16, 128>(a, p, s, ev);
    return attn_launch_t<bf16, 64>(a, p, s, ev);
  }
  if (a.hd == 128) return attn_launch_t<float, 128>(a, p, s, ev);
  return attn_launch_t<float, 64>(a, p, s, ev);
}

}  // namespace dv
