/*
 * deltavision.h - C ABI of the MI355X (gfx950) visual-memory library.
 *
 * The library implements the hot path of delta-Vision ("Just MLPs: Efficient
 * Visual State Reconstruction for Multimodal Language Models"): per-layer
 * low-rank adapters build each layer's visual memory from the shared visual
 * embeddings (Section 3.1, Eq. 4-5), the memory is normalised and projected by
 * the frozen per-layer key/value weights (Section 3.2, Eq. 7), and text queries
 * attend over all visual keys plus their own causal text context (Section 3.2,
 * Eq. 9). Visual tokens never get queries, attention outputs or FFN updates.
 *
 * Conventions shared by every call
 *  - Pointers are DEVICE pointers to dense, row-major tensors in the shapes
 *    given below, 16-byte aligned. Outputs must not alias inputs.
 *  - `dtype` (dv_dtype) applies to every tensor of a call, including Z and the
 *    workspace-backed intermediates. Accumulation is always fp32.
 *  - Weights are stored out x in, like nn.Linear: Dw[l] = D_l^T [r,d],
 *    Uw[l] = U_l^T [d,r], Wk[l], Wv[l] [Hkv*hd, d].
 *  - `stream` is a hipStream_t (NULL = the default stream). Every call only
 *    enqueues work on it and returns; nothing is synchronised.
 *  - Ownership: the caller allocates and frees every buffer, including the
 *    workspace. The library keeps no state besides a thread-local error text
 *    and the thread-local events of the profiling hook (dv_time_kernel).
 *  - Errors: arguments are validated on the host before anything is enqueued;
 *    on error nothing is launched and no output is written. A failed launch
 *    returns DV_ERR_HIP. No C++ exception crosses this boundary.
 *  - Debugging: with DV_DEBUG set (to anything but "0") in the environment, every
 *    call waits for the kernels it enqueued and returns DV_ERR_HIP if one of them
 *    failed (e.g. a memory fault), so the failing call is the one that reports it.
 *    It synchronises the stream, so it is not for streams under graph capture.
 *  - Supported: dtype f32 or bf16; hd in {64, 128}; Hq % Hkv == 0;
 *    d % 64 == 0; r % 16 == 0; all sizes > 0 unless stated.
 */
#ifndef DELTAVISION_H_
#define DELTAVISION_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  DV_OK = 0,
  DV_ERR_NULL = 1,        /* a required pointer is NULL */
  DV_ERR_SHAPE = 2,       /* sizes are negative, zero where not allowed, or inconsistent */
  DV_ERR_UNSUPPORTED = 3, /* valid but outside the supported set (dtype, act, hd, d, r) */
  DV_ERR_ALIGN = 4,       /* a pointer is not 16-byte aligned */
  DV_ERR_WORKSPACE = 5,   /* workspace NULL or smaller than the minimum */
  DV_ERR_HIP = 6,         /* the HIP runtime reported an error while enqueuing */
  DV_ERR_INTERNAL = 7
} dv_status;

typedef enum { DV_F32 = 0, DV_BF16 = 1 } dv_dtype;

typedef enum {
  DV_ACT_SILU = 0, /* phi of Section 3.1 */
  DV_ACT_GELU = 1  /* x * Phi(x), exact (erf) form */
} dv_act;

/*
 * Down half of the adapter (Section 3.1, Eq. 4) for ALL layers at once. The
 * embedding adapter (Eq. 5) feeds every layer the same E, so the per-layer
 * products E D_l form one GEMM of E against [D_0 | ... | D_{L-1}]:
 *     Z[l][t][j] = phi( sum_k E[t][k] * Dw[l][j][k] ),   l < L, t < T, j < r.
 *   E  [T, d]     visual embeddings (Section 2, Eq. 1), T = batch * visual tokens
 *   Dw [L, r, d]  down-projections, out x in
 *   Z  [L, T, r]  output (dtype of the call), phi applied in fp32 before rounding
 *   act           dv_act
 */
dv_status dv_build_visual_memory(const void* E, const void* Dw, void* Z, int64_t T, int32_t d,
                                 int32_t L, int32_t r, int32_t act, int32_t dtype, void* stream);

/*
 * Up half of the adapter (Eq. 4-5) and the visual key/value projection
 * (Section 3.2, Eq. 7) for layers l0 <= l < l0 + nl:
 *     M_l  = E + Z_l U_l                       (memory of layer l)
 *     N_l  = M_l * rsqrt(mean_k M_l^2 + eps) * gamma_l   (LN_l read as RMSNorm)
 *     Kv_l = N_l Wk[l]^T,  Vv_l = N_l Wv[l]^T, stored head-major
 *   E     [B*Nv, d]
 *   Z     [L, B*Nv, r]   from dv_build_visual_memory
 *   Uw    [L, d, r]      up-projections, out x in
 *   gamma [L, d]         frozen RMSNorm weights
 *   Wk,Wv [L, Hkv*hd, d] frozen key / value projections
 *   Kv,Vv [L, B, Hkv, Nv, hd] outputs; only the slots of layers l0..l0+nl-1 are written
 *   ws    workspace; at least dv_project_visual_kv_workspace(B*Nv, d, 1, dtype) bytes.
 *         With room for k layers the call processes layers in groups of up to k;
 *         dv_project_visual_kv_workspace(B*Nv, d, nl, dtype) holds all of them at once.
 * M_l is transient (it lives only in the workspace), as the method prescribes.
 * Narrow K/V widths can take one fused kernel instead (dv_set_fused_kv): it keeps M_l of 64
 * tokens on chip and projects it at once, so the workspace is validated but not used. Its
 * rounding points are the same (M_l in fp32, M_l * gamma_l rounded to the call dtype before the
 * projection, the row scale applied to the fp32 product); only the order in which the row sum
 * of squares and the products over d are added up differs.
 */
size_t dv_project_visual_kv_workspace(int64_t T, int32_t d, int32_t nl, int32_t dtype);
dv_status dv_project_visual_kv(const void* E, const void* Z, const void* Uw, const void* gamma,
                               const void* Wk, const void* Wv, void* Kv, void* Vv, int32_t B,
                               int32_t Nv, int32_t d, int32_t L, int32_t r, int32_t Hkv,
                               int32_t hd, int32_t l0, int32_t nl, float eps, int32_t dtype,
                               void* ws, size_t ws_bytes, void* stream);

/*
 * Fused up-projection + RMSNorm + K/V kernel for narrow K/V widths: bf16, 2 * Hkv * hd = 1024
 * (e.g. 4 K/V heads of 128), r in {128, 256, 512}, d a multiple of 64. The 64 x 1024 fp32 K/V
 * accumulators of a block fit in registers, so M_l is computed once per token and never
 * written out. It is off by default: each block of 64 tokens reads the layer's whole U_l and
 * [Wk | Wv] from the L2, about 1.4 times the L2-to-CU traffic of the two-kernel path, and on
 * MI355X at the Qwen2.5-VL video shape it measured slower than that path despite saving the
 * workspace round trip.
 *   dv_set_fused_kv(1) makes dv_project_visual_kv, dv_project_visual_kv_ex with no epilogue
 *   step and dv_kept_visual_kv take it for those sizes; dv_set_fused_kv(0) restores the
 *   default. Process-wide; a call already enqueued keeps its kernel. on must be 0 or 1.
 *   dv_project_visual_kv_fused returns 1 when a call with these sizes takes the fused kernel
 *   under the current setting, else 0 (also for any size the projection rejects); no GPU work.
 */
dv_status dv_set_fused_kv(int32_t on);
int32_t dv_project_visual_kv_fused(int32_t d, int32_t r, int32_t Hkv, int32_t hd, int32_t dtype);

/*
 * Kernel for M_l * gamma_l and the row sums of squares in the bf16 projection (dv_project_visual_kv,
 * dv_project_visual_kv_ex, dv_kept_visual_kv); both compute Eq. 5 and the RMSNorm statistics of
 * Eq. 7 with the same products in the same order, so M_l * gamma_l is the same to the bit and
 * only the order in which the row sum of squares is added up differs.
 *   1 (tiled): each block computes a 128 x 128 tile of M_l for up to four layers.
 *   2 (Z-resident): each block takes 128 rows of one layer, keeps their Z_l in registers and
 *     walks all of d, streaming only U_l; for r = 256 or 512 (other ranks take the tiled kernel).
 *   0 (default): the Z-resident kernel where r is 256 and there are at least eight rounds
 *     (2048) of its blocks (ceil(B*Nv / 128) * nl), else the tiled kernel.
 * dv_set_up_kernel(mode) selects, process-wide (a call already enqueued keeps its kernel);
 * mode must be 0, 1 or 2. dv_project_visual_kv_up_kernel returns the kernel (1 or 2) a bf16 call
 * with these sizes takes under the current setting, 1 for any other dtype; no GPU work.
 */
dv_status dv_set_up_kernel(int32_t mode);
int32_t dv_project_visual_kv_up_kernel(int64_t T, int32_t d, int32_t r, int32_t nl, int32_t dtype);

/*
 * Recurrent adapter (Section 3.1, Eq. 6) and the visual K/V projection (Section 3.2, Eq. 7) of
 * every layer in one call:
 *     M_{-1} = E,   M_l = M_{l-1} + phi(M_{l-1} D_l) U_l,   l = 0 .. L-1,
 *     Kv_l, Vv_l = RMSNorm(M_l; gamma_l, eps) Wk[l]^T, ... Wv[l]^T   (head-major, as above).
 * Layer l's down projection needs layer l-1's memory, so the layers run in order; the
 * layer-to-layer state is kept in fp32 in the workspace for both dtypes.
 *   E, Dw, Uw, gamma, Wk, Wv, Kv, Vv   as for dv_build_visual_memory / dv_project_visual_kv
 *   act   dv_act
 *   ws    at least dv_recurrent_visual_kv_workspace(B*Nv, d, L, r, dtype) bytes
 */
size_t dv_recurrent_visual_kv_workspace(int64_t T, int32_t d, int32_t L, int32_t r, int32_t dtype);
dv_status dv_recurrent_visual_kv(const void* E, const void* Dw, const void* Uw, const void* gamma,
                                 const void* Wk, const void* Wv, void* Kv, void* Vv, int32_t B,
                                 int32_t Nv, int32_t d, int32_t L, int32_t r, int32_t Hkv,
                                 int32_t hd, int32_t act, float eps, int32_t dtype, void* ws,
                                 size_t ws_bytes, void* stream);

/*
 * Backbone epilogue of the visual K/V (outside Eq. 7). The paper keeps every visual token at
 * its original position (appendix on hidden-state compression), so a backbone that adds a
 * bias to its K/V projections, normalises each key head or rotates keys by position does the
 * same to the reconstructed visual K/V, in this order, for layer l, token (b, i), head h:
 *   K += k_bias[l],  V += v_bias[l]
 *   K_h <- K_h * (mean_c K_h[c]^2 + k_norm_eps)^-1/2 * k_norm[l]      (per-head key RMSNorm)
 *   rotary embedding of K_h: channel j < hd/2 pairs with channel j + hd/2 and turns by the
 *   angle p * rope_theta^(-2j/hd), p = positions[b][a][i], where the position axis a is 0
 *   for j < rope_sections[0], 1 for j < rope_sections[0] + rope_sections[1], 2 otherwise
 *   (multimodal rotary sections; {hd/2, 0, 0} is the one-dimensional rotation):
 *       (k_j, k_{j+hd/2}) <- (k_j cos - k_{j+hd/2} sin,  k_{j+hd/2} cos + k_j sin).
 * A NULL k_bias, v_bias, k_norm or positions skips its step. bf16 runs round the projection
 * to bf16 once before the key norm and the rotation (with the bias included when r is a
 * multiple of 64, before it otherwise) and the result once more at the end.
 */
typedef struct {
  const void* k_bias;        /* [L, Hkv*hd] in the call dtype, 16-byte aligned, or NULL */
  const void* v_bias;        /* [L, Hkv*hd] in the call dtype, 16-byte aligned, or NULL */
  const void* k_norm;        /* [L, hd] in the call dtype, 16-byte aligned, or NULL */
  float k_norm_eps;          /* finite, >= 0 */
  const int32_t* positions;  /* device [B, 3, Nv] position ids per axis, or NULL: no rotation */
  int32_t rope_sections[3];  /* non-negative, adding up to hd/2 (read only with positions) */
  float rope_theta;          /* finite, > 0 (read only with positions) */
} dv_kv_epilogue;

/*
 * dv_project_visual_kv followed by the backbone epilogue above (fused into the bf16 K/V
 * kernel). epi may be NULL (then identical to dv_project_visual_kv). ws holds the rotary
 * table (T * hd * 4 bytes, 256-aligned) followed by the projection workspace: at least
 * dv_project_visual_kv_ex_workspace(B*Nv, d, 1, hd, dtype) bytes;
 * dv_project_visual_kv_ex_workspace(B*Nv, d, nl, hd, dtype) bytes project all nl layers in one
 * launch.
 */
size_t dv_project_visual_kv_ex_workspace(int64_t T, int32_t d, int32_t nl, int32_t hd,
                                         int32_t dtype);
dv_status dv_project_visual_kv_ex(const void* E, const void* Z, const void* Uw, const void* gamma,
                                  const void* Wk, const void* Wv, void* Kv, void* Vv, int32_t B,
                                  int32_t Nv, int32_t d, int32_t L, int32_t r, int32_t Hkv,
                                  int32_t hd, int32_t l0, int32_t nl, float eps,
                                  const dv_kv_epilogue* epi, int32_t dtype, void* ws,
                                  size_t ws_bytes, void* stream);

/*
 * Layer-wise adapter skipping (appendix on adapter skipping, Tables 14 and 15): the
 * embedding adapter (Eq. 4-5) and the K/V projection (Eq. 7) run only for the layers
 * with keep[l] != 0. A skipped layer gets no visual keys at all (its attention runs
 * with Nv = 0, the text-only case of Eq. 18), so the caches hold only the kept layers,
 * packed in layer order: cache slot j is the j-th kept layer.
 *   keep    HOST array of L bytes (not device memory), read during the call only
 *   E, Dw, Uw, gamma, Wk, Wv   full L-layer weights as for dv_build_visual_memory /
 *           dv_project_visual_kv
 *   Kv, Vv  [nkeep, B, Hkv, Nv, hd], nkeep = number of nonzero keep bytes; may be
 *           NULL when nkeep == 0 (then nothing is launched and DV_OK is returned)
 *   ws      holds Z of the kept layers plus the projection workspace: at least
 *           dv_kept_visual_kv_workspace(B*Nv, d, r, 1, dtype) bytes; with
 *           dv_kept_visual_kv_workspace(B*Nv, d, r, nkeep, dtype) bytes every kept layer
 *           is projected in one launch per contiguous run of kept layers.
 * Kept layer l gives bit-identical K/V to dv_project_visual_kv for that layer (same
 * kernels, same arithmetic order).
 */
size_t dv_kept_visual_kv_workspace(int64_t T, int32_t d, int32_t r, int32_t nkeep, int32_t dtype);
dv_status dv_kept_visual_kv(const void* E, const void* Dw, const void* Uw, const void* gamma,
                            const void* Wk, const void* Wv, const uint8_t* keep, void* Kv,
                            void* Vv, int32_t B, int32_t Nv, int32_t d, int32_t L, int32_t r,
                            int32_t Hkv, int32_t hd, int32_t act, float eps, int32_t dtype,
                            void* ws, size_t ws_bytes, void* stream);

/*
 * Text-query attention of one layer over [visual; text] keys (Section 3.2,
 * Eq. 9; visual tokens precede the text, Section 2 Eq. 2):
 *     O[b,i,h,:] = sum_j softmax_j( scale * <Q[b,i,h,:], K_j> ) V_j
 * over every visual key j < Nv of kv-head g = h / (Hq/Hkv) and the text keys
 * 0..q_pos0+i of the same head (causal). Prefill: q_pos0 = 0, Nq = Nkt. Decode:
 * Nq = 1 and q_pos0 = number of earlier text tokens (the new token's key is
 * text key q_pos0). Nv may be 0 (visual read blocked).
 *   Q, O   [B, Nq, Hq, hd]
 *   Kv, Vv [B, Hkv, Nv, hd]   one layer of the visual cache (may be NULL when Nv == 0)
 *   Kt, Vt [B, Hkv, Nkt, hd]  text key / value cache; requires q_pos0 + Nq <= Nkt (text keys
 *          past q_pos0 + Nq - 1, e.g. the free slots of a preallocated cache, are never read)
 *   Sizes: one (batch, kv-head) slice of either cache holds at most 2^31-1 bytes
 *          (Nv*hd*elem_size and Nkt*hd*elem_size), otherwise DV_ERR_SHAPE
 *   scale  softmax scale, finite and > 0, usually 1/sqrt(hd)
 *   ws     split-key partials; may be NULL/0 (then keys are not split). With
 *          dv_text_visual_attention_workspace(...) bytes the call picks its
 *          preferred split; with fewer it uses the largest split that fits.
 */
size_t dv_text_visual_attention_workspace(int32_t B, int32_t Hq, int32_t Hkv, int32_t hd,
                                          int32_t Nv, int32_t Nq, int32_t Nkt);
dv_status dv_text_visual_attention(const void* Q, const void* Kv, const void* Vv, const void* Kt,
                                   const void* Vt, void* O, int32_t B, int32_t Hq, int32_t Hkv,
                                   int32_t hd, int32_t Nv, int32_t Nq, int32_t Nkt,
                                   int32_t q_pos0, float scale, int32_t dtype, void* ws,
                                   size_t ws_bytes, void* stream);

/*
 * dv_text_visual_attention for callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc). Same arguments, same result
 * bits as dv_text_visual_attention with its recommended workspace, but the key-split partials
 * live in a static array of DV_ATTENTION_SCRATCH_BYTES inside the library: each GPU the library
 * runs on holds its own copy until the process ends. The call allocates and frees nothing and
 * clears nothing (every partial is written before it is read). A call whose key split needs
 * more partials than the array holds returns DV_ERR_WORKSPACE without launching (the
 * LLaVA-NeXT-sized prefill, 8 x 128 queries x 32 heads over 2880 visual keys, is one); such
 * calls go through dv_text_visual_attention with a workspace.
 * All calls on one GPU share its array: calls that may overlap on one GPU (different streams,
 * or different threads without ordering) race on it and must be serialised by the caller.
 * The stream must belong to the current device.
 */
#define DV_ATTENTION_SCRATCH_BYTES ((size_t)32 << 20)
dv_status dv_text_visual_attention_noalloc(const void* Q, const void* Kv, const void* Vv,
                                           const void* Kt, const void* Vt, void* O, int32_t B,
                                           int32_t Hq, int32_t Hkv, int32_t hd, int32_t Nv,
                                           int32_t Nq, int32_t Nkt, int32_t q_pos0, float scale,
                                           int32_t dtype, void* stream);

/*
 * Visual write into a linear-attention (Gated DeltaNet) recurrent state (appendix on linear
 * attention, Eq. 15-16): for every sequence b and value head h, the visual tokens t = 0..N-1
 * are written in order,
 *     S <- alpha_t S,   then   S <- S + beta_t k_t (v_t - S^T k_t)^T,
 * where value head h uses key head h / (Hv/Hk). k, v, alpha and beta come from the backbone's
 * own norm, projections, causal convolution and gates applied to the visual memories; only
 * the final state is produced (visual positions take the next layer's memory instead of the
 * layer outputs).
 *   k      [B, Hk, N, dk]  call dtype
 *   v      [B, Hv, N, dv]  call dtype
 *   alpha  [B, Hv, N]      fp32 gates in (0, 1] (values <= 0 act as the smallest positive float)
 *   beta   [B, Hv, N]      fp32 write strengths
 *   S      [B, Hv, dk, dv] fp32 state, read and overwritten in place
 *   dk, dv in {64, 128}; N may be 0 (nothing is launched)
 *   ws     at least dv_delta_rule_workspace(B, Hv, N, dk, dv, dtype) bytes
 * Chunks of 64 tokens are prepared in parallel and then applied in order; the products with
 * the state read it rounded to the call dtype while the state itself stays fp32.
 */
size_t dv_delta_rule_workspace(int32_t B, int32_t Hv, int32_t N, int32_t dk, int32_t dv,
                               int32_t dtype);
dv_status dv_delta_rule_write(const void* k, const void* v, const float* alpha, const float* beta,
                              float* S, int32_t B, int32_t Hk, int32_t Hv, int32_t N, int32_t dk,
                              int32_t dv, int32_t dtype, void* ws, size_t ws_bytes, void* stream);

/*
 * Profiling hook. Kernels of the library, as named by dv_kernel:
 *   DV_KERNEL_DOWN       the all-layer down-projection of dv_build_visual_memory, or the
 *                        whole per-layer adapter chain of dv_recurrent_visual_kv
 *   DV_KERNEL_UP         the up-projection + residual of dv_project_visual_kv
 *   DV_KERNEL_KV         the RMSNorm-scaled K/V projection of dv_project_visual_kv and
 *                        dv_recurrent_visual_kv; when dv_project_visual_kv takes the fused
 *                        kernel, that kernel, which also does the up-projection
 *                        (DV_KERNEL_UP then records nothing)
 *   DV_KERNEL_ATTENTION  the main attention kernel of dv_text_visual_attention
 *                        (without the split-merge kernel)
 *   DV_KERNEL_DELTA_PREP the per-chunk preparation of dv_delta_rule_write
 *   DV_KERNEL_DELTA_SCAN the in-order chunk chain of dv_delta_rule_write (with the segment merge
 *                        when the sequence is split into segments)
 * After dv_time_kernel(k, begin, end) with two hipEvent_t handles, every launch
 * of kernel k made by later calls on this thread is bracketed by
 * hipEventRecord(begin) and hipEventRecord(end) on the call's stream; when a
 * call launches k several times (a projection in layer groups) the pair spans
 * the first to the last launch. NULL, NULL switches the hook off. The events
 * stay owned by the caller and must outlive the calls that record them.
 */
typedef enum {
  DV_KERNEL_DOWN = 0,
  DV_KERNEL_UP = 1,
  DV_KERNEL_KV = 2,
  DV_KERNEL_ATTENTION = 3,
  DV_KERNEL_DELTA_PREP = 4,
  DV_KERNEL_DELTA_SCAN = 5
} dv_kernel;
dv_status dv_time_kernel(int32_t kernel, void* ev_begin, void* ev_end);

/* Measurement probe, not part of the method: the sustained bf16 MFMA rate of this GPU. The
 * chip's clock drops under MFMA load, and drops further the more the operand bits toggle, so the
 * rate a GEMM can reach depends on its data. The probe enqueues 1024 blocks of 8 waves; each wave
 * issues iters x 32 independent v_mfma_f32_16x16x32_bf16 (the instruction of the build GEMMs) on
 * register operands, with no memory traffic, and block b writes one float to sink[b].
 *   random  != 0: operands are random bf16 bit patterns (spread exponents, random mantissas);
 *           0: constant operands.
 *   iters   in [1, 1 << 20]; the call performs 1024 * 8 * iters * 32 * 16384 FLOP.
 *   sink    device memory of at least 1024 floats, caller-owned, 16-byte aligned.
 * Time it with events on `stream` around the call. */
dv_status dv_probe_mfma(int32_t random, int32_t iters, float* sink, void* stream);

/* Human-readable name of a status code (static storage). */
const char* dv_status_string(int32_t status);
/* Detail of the last error raised on the calling thread ("" if none). */
const char* dv_last_error(void);
/* ABI version, incremented on any incompatible change. */
int32_t dv_abi_version(void);

#ifdef __cplusplus
}
#endif

#endif /* DELTAVISION_H_ */
