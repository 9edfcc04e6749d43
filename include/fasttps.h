/*
 * fasttps.h -- C ABI of the FastTPS token-phase decoder layer for MI355X (gfx950).
 *
 * One call of fasttps_decode_step runs one decode step of one pre-norm decoder
 * layer for B sequences, each holding one new token (the token phase of the
 * FastTPS paper, Section 2.1: B x N x D activations with N = 1):
 *
 *   h  = RMSNorm1(x)                              (Section 2.3 step 1, Alg. 4)
 *   q, k, v = W_q h, W_k h, W_v h                 (Section 2.2)
 *   q, k = RoPE(q, k) at position N_p             (Alg. 3, joint RoPE; Eq. 22)
 *   K_cache[b, g, N_p] = bf16(k), V_cache[b, g, N_p] = bf16(v)
 *                                                 (GKVC in-place append, Eq. 1)
 *   o  = softmax(q K^T / sqrt(d)) V over the N_p + 1 entries  (Eq. 25-28)
 *   h1 = x + W_o o
 *   y  = h1 + W_down (SiLU(W_gate h2) * (W_up h2)),  h2 = RMSNorm2(h1)
 *                                                 (Eq. mlp_main; Alg. 4, Eq. 29-32)
 *
 * Conventions
 *   - Tensors are bfloat16 (bit patterns in uint16 storage) unless stated.
 *   - "device" pointers are HIP device addresses on the current device;
 *     "host" pointers are ordinary CPU memory.
 *   - Weight matrices use the [out, in] row-major layout of nn.Linear.
 *   - Caches are [B_max, H_kv, N_max, d] row-major, contiguous; the slot of
 *     (b, g, n) is at element ((b * H_kv + g) * N_max + n) * d  (Eq. 1 with
 *     N_p + N_r = N_max).
 *   - Every function returns FASTTPS_OK (0) or a negative status. No
 *     exception or abort crosses the ABI. All argument checks happen before
 *     the first HIP call, so a rejected call has no side effect. The text of
 *     the last error on the calling thread is given by fasttps_last_error().
 *   - Streams are hipStream_t passed as void*; NULL means the default stream.
 */
#ifndef FASTTPS_H
#define FASTTPS_H

#include <stddef.h>
#include <stdint.h>

#if defined(__GNUC__) || defined(__clang__)
#define FASTTPS_API __attribute__((visibility("default")))
#else
#define FASTTPS_API
#endif

#ifdef __cplusplus
extern "C" {
#endif

/* ---- status codes ---------------------------------------------------- */
#define FASTTPS_OK                0
#define FASTTPS_ERR_INVALID_ARG  -1  /* null pointer, size out of range, overlap */
#define FASTTPS_ERR_UNSUPPORTED  -2  /* shape the kernels are not built for */
#define FASTTPS_ERR_ALIGNMENT    -3  /* a tensor pointer is not 16-byte aligned */
#define FASTTPS_ERR_CACHE_FULL   -4  /* some pos[b] >= N_max (N_r = 0) or pos[b] < 0 */
#define FASTTPS_ERR_OOM          -5  /* device allocation failed */
#define FASTTPS_ERR_HIP          -6  /* a HIP runtime call failed (text in last_error) */
#define FASTTPS_ERR_BAD_HANDLE   -7  /* handle null, destroyed, or of another layer */

typedef struct fasttps_layer fasttps_layer;      /* config, scratch, RoPE table */
typedef struct fasttps_weights fasttps_weights;  /* packed weights of one layer */

/* Shape of one decoder layer. */
typedef struct {
  int32_t hidden;        /* D; multiple of 8, 8 <= D <= 8192 */
  int32_t n_heads;       /* H query heads; H / H_kv in {1, 2, 4}; H * d <= 8192 */
  int32_t n_kv_heads;    /* H_kv */
  int32_t head_dim;      /* d in {64, 96, 128} */
  int32_t intermediate;  /* K (MLP width); multiple of 8, <= 32768 */
  int32_t max_batch;     /* B_max in [1, 64] */
  int32_t max_seq;       /* N_max = N_p + N_r: cache capacity per sequence (Eq. 1), >= 1 */
  float rope_base;       /* RoPE base (e.g. 1e4, 5e5); angle_j(n) = n * base^(-2j/d) */
  float rms_eps;         /* RMSNorm epsilon, added inside the square root, > 0 */
} fasttps_config;

/* Raw weights of one layer: device pointers, bf16, nn.Linear layout. */
typedef struct {
  const void* attn_norm;  /* [D]        gain of RMSNorm1 */
  const void* w_q;        /* [H*d, D]   */
  const void* w_k;        /* [H_kv*d, D] */
  const void* w_v;        /* [H_kv*d, D] */
  const void* w_o;        /* [D, H*d]   */
  const void* mlp_norm;   /* [D]        gain of RMSNorm2 */
  const void* w_gate;     /* [K, D]     */
  const void* w_up;       /* [K, D]     */
  const void* w_down;     /* [D, K]     */
} fasttps_weights_desc;

/* Create a layer handle on the current device: validates the config,
 * allocates the step's scratch (sized for max_batch) and builds the RoPE
 * cos/sin table for positions [0, N_max) (computed in double precision on the
 * host; the paper feeds sin/cos to RoPE as inputs, Alg. 1 and Alg. 3).
 * The handle owns its memory until fasttps_layer_destroy. Blocking. */
FASTTPS_API int fasttps_layer_create(const fasttps_config* cfg, fasttps_layer** out);

/* Pack one layer's raw weights into the library's layout: fused [W_q; W_k;
 * W_v] rows, interlaced gate/up rows (Section 3.2 item 1, Alg. 4: tiles of
 * gate rows alternate with the matching up rows) and W_down as given
 * ([D, K], one contiguous K-row per output). Runs on `stream` and
 * returns once the copies are complete; the raw weights may then be freed.
 * The packed weights belong to the returned handle (free with
 * fasttps_weights_free) and may be used with any layer handle of the same
 * config. */
FASTTPS_API int fasttps_weights_pack(fasttps_layer* layer, const fasttps_weights_desc* w,
                         void* stream, fasttps_weights** out);

/* One decode step (see the top of this file).
 *   x        device, [batch, D] bf16 input token activations
 *   pos      host, [batch] int32: N_p of each sequence = index of the new
 *            token = number of valid cache entries before the call
 *   batch    number of sequences, 1 <= batch <= max_batch
 *   k_cache, v_cache
 *            device, [batch, H_kv, N_max, d] bf16 (a leading block of a
 *            [B_max, ...] cache is fine). Entries [0, pos[b]) are read; the
 *            one slot pos[b] of every (b, g) is written; nothing else is
 *            written. Nothing else is read either, with one exception: a
 *            sequence with pos[b] = 0 has no cached entry, and the attention's
 *            loads, issued ahead of their use and clamped to entry
 *            max(pos[b] - 1, 0), then read slot 0 before or while it is being
 *            written and discard the values. After the call the caller's
 *            length is pos[b] + 1 (Section 3.1.1 GKVC: N_p <- N_p + 1,
 *            N_r <- N_r - 1).
 *   y        device, [batch, D] bf16 output; must not overlap x or the caches
 *   stream   the step is enqueued on this stream; the call neither allocates
 *            nor synchronizes.
 * All tensors must be 16-byte aligned. A handle's scratch is shared by its
 * calls, so steps on one handle must not run concurrently on different
 * streams. */
FASTTPS_API int fasttps_decode_step(fasttps_layer* layer, const fasttps_weights* w, const void* x,
                        const int32_t* pos, int32_t batch, void* k_cache, void* v_cache,
                        void* y, void* stream);

/* fasttps_decode_step for callers that cannot allocate (code under HIP
 * graph capture, tight serving loops, harnesses that forbid hipMalloc): the
 * same arguments, checks, cache contract and results, computed by the same
 * vector-path kernels (whatever fasttps_set_gemm_path says), with the step's
 * fp32 intermediates in a static device array of the library (8 MiB per
 * device, held until the process ends) instead of the handle's scratch. The
 * call allocates nothing. Returns FASTTPS_ERR_UNSUPPORTED, before any
 * launch, when the step's intermediates (q|k|v, the attention's split
 * partials, o, h1 and the MLP activation, each 256-byte aligned, for `batch`
 * sequences) exceed 8 MiB; the five workloads of this library need at most
 * about 3 MiB (16 sequences of the Phi-3-mini layer). Every call on a device
 * shares that device's array and overwrites it, so calls on one device
 * whose executions overlap (different streams, or threads) race; the test
 * hooks (fasttps_debug_read, fasttps_profile_*) do not see these steps. */
FASTTPS_API int fasttps_decode_step_noalloc(fasttps_layer* layer, const fasttps_weights* w, const void* x,
                                            const int32_t* pos, int32_t batch, void* k_cache, void* v_cache,
                                            void* y, void* stream);

/* 8-bit KV cache formats for fasttps_decode_step_kv8. */
#define FASTTPS_KV_FP8_E4M3 1 /* OCP E4M3: bias 7, subnormals, largest finite 448, 0x7F/0xFF NaN */
#define FASTTPS_KV_INT8 2     /* two's complement, entries in [-127, 127] */

/* One decode step over an 8-bit KV cache. The paper holds its cache layout
 * and append compatible with a quantized cache (Section 5.2, Compatibility
 * with Acceleration Algorithm; Section 2.4, Operator Type and OI, counts the
 * quantized cache's concatenation among the memory reorganisation
 * operators) without fixing a format; this is the reading implemented:
 *   kv_format  FASTTPS_KV_FP8_E4M3 or FASTTPS_KV_INT8
 *   k_cache, v_cache
 *              device, [batch, H_kv, N_max, d] of 8-bit codes, the GKVC layout
 *              of Eq. 1 with one byte per element (16-byte aligned). An entry
 *              of KV head g means k_scale[g] * value(code) (v_scale[g] for V).
 *   k_scale, v_scale
 *              host, [H_kv] float: the per-KV-head scales, positive and
 *              finite; they are copied into the launch, so a captured graph
 *              keeps the values of the call that was captured.
 * The new entry of each (b, g) is rounded once, in double precision, to the
 * nearest code of k_rope / k_scale[g] (v / v_scale[g]), ties to the even
 * code, magnitudes beyond the largest finite value saturating to it (448 or
 * 127), and written to slot pos[b]; attention uses that rounded entry. The
 * other arguments, the cache contract and the errors are those of
 * fasttps_decode_step; in addition FASTTPS_ERR_INVALID_ARG for an unknown
 * format or a scale that is not positive and finite. */
FASTTPS_API int fasttps_decode_step_kv8(fasttps_layer* layer, const fasttps_weights* w, const void* x,
                            const int32_t* pos, int32_t batch, int32_t kv_format, void* k_cache,
                            void* v_cache, const float* k_scale, const float* v_scale, void* y,
                            void* stream);

/* The op-by-op baseline: the same step computed the way the paper's
 * standard implementation does it (Alg. 1: RoPE, Transpose, Concat, QK^T,
 * Softmax, PV; Alg. 2: gate, SiLU, up, elementwise mul, down; RMSNorm, the
 * separate Q, K, V, O projections and the residual adds as operators of
 * their own), each operator a kernel whose inputs and outputs go through
 * HBM, and the Concat rebuilding each sequence's K and V cache in a new
 * buffer (the cache reload that GKVC removes, Section 3.1.1). It exists to
 * measure the fused step against. Same arguments, results (within the same
 * tolerances) and cache contract as fasttps_decode_step: slot pos[b] of the
 * caller's caches is written, nothing else of them. Needs the baseline's
 * scratch, allocated once per layer handle by fasttps_unfused_enable
 * (blocking; about 2 B H_kv N_max d bf16 plus the fp32 intermediates, for
 * max_batch sequences; freed with the layer). Returns FASTTPS_ERR_INVALID_ARG
 * if the scratch was not enabled. */
FASTTPS_API int fasttps_unfused_enable(fasttps_layer* layer);
FASTTPS_API int fasttps_decode_step_unfused(fasttps_layer* layer, const fasttps_weights* w, const void* x,
                                const int32_t* pos, int32_t batch, void* k_cache, void* v_cache,
                                void* y, void* stream);

/* Which kernels run the four projections (QKV, O, gate/up, down).
 *   FASTTPS_GEMM_VECTOR  weight-streaming GEMVs on the vector ALUs (fp32
 *                        activations); the only path of a layer with
 *                        max_batch == 1
 *   FASTTPS_GEMM_MATRIX  weight-streaming MFMA kernels (bf16 weights times
 *                        activations split into two bf16 levels, fp32
 *                        accumulation); needs max_batch > 1, for which
 *                        fasttps_weights_pack also stores the weights in the
 *                        MFMA tile order (about twice the weight memory, or
 *                        the tiles only: fasttps_set_weight_layout)
 *   FASTTPS_GEMM_FUSED   one sequence in one persistent kernel (below); a
 *                        measured alternative, slower on MI355X than the
 *                        separate kernels of the vector path replayed from a
 *                        HIP graph
 *   FASTTPS_GEMM_AUTO    (default) the matrix path from 2 sequences up where
 *                        the weights carry the tiles, else the vector path
 * At batch 8-16 the projections are dense enough that the multiply-adds
 * outgrow the vector ALUs beside the weight stream (Section 4.4, OI and Accuracy, puts the
 * token-phase projections at the weight stream); both paths read every
 * weight once per step. Returns FASTTPS_ERR_INVALID_ARG for an unknown path,
 * or for FASTTPS_GEMM_MATRIX on a layer with max_batch == 1. A step with the
 * matrix path and weights packed for max_batch == 1 fails with
 * FASTTPS_ERR_INVALID_ARG before any launch. */
#define FASTTPS_GEMM_AUTO 0
#define FASTTPS_GEMM_VECTOR 1
#define FASTTPS_GEMM_MATRIX 2
#define FASTTPS_GEMM_FUSED 3  /* one sequence: the whole step as one persistent kernel
                                 (the vector GEMVs and the attention as phases of one
                                 launch); shapes it is built for, else the step fails
                                 with FASTTPS_ERR_UNSUPPORTED before any launch */
FASTTPS_API int fasttps_set_gemm_path(fasttps_layer* layer, int32_t path);

/* How fasttps_weights_pack stores the four projections for a layer with
 * max_batch > 1 (a layer with max_batch == 1 stores them row-major only).
 *   FASTTPS_WEIGHTS_ROWS_AND_TILES
 *                        (default) row-major for the vector path and in the
 *                        MFMA tile order for the matrix path: twice the
 *                        projection memory (Phi-3-mini: 453 instead of 227 MB
 *                        per layer), so that steps of one sequence keep the
 *                        vector kernels, the faster ones at batch 1 (Phi-3
 *                        layer at KV 4096 on MI355X: 59.9 against 68.0 us per
 *                        layer step on the matrix path)
 *   FASTTPS_WEIGHTS_TILES
 *                        the tile order only: every step with these weights
 *                        runs the matrix path, also at one sequence; steps
 *                        that need row-major weights (FASTTPS_GEMM_VECTOR or
 *                        FASTTPS_GEMM_FUSED set, FASTTPS_MLP_FUSED set,
 *                        fasttps_decode_step_noalloc,
 *                        fasttps_decode_step_unfused) fail with
 *                        FASTTPS_ERR_INVALID_ARG before any launch, and so
 *                        does a pack with FASTTPS_MLP_FUSED selected.
 * Applies to weights packed afterwards with this handle (the pack then
 * allocates and frees a temporary row-major copy of W_q|W_k|W_v). Returns
 * FASTTPS_ERR_INVALID_ARG for an unknown layout, or for FASTTPS_WEIGHTS_TILES
 * on a layer with max_batch == 1. */
#define FASTTPS_WEIGHTS_ROWS_AND_TILES 0
#define FASTTPS_WEIGHTS_TILES 1
FASTTPS_API int fasttps_set_weight_layout(fasttps_layer* layer, int32_t layout);

/* How the MLP (RMSNorm2, gate/up, siLu_Mul, down, residual) runs.
 *   FASTTPS_MLP_SPLIT  (default) two kernels: gate/up with siLu_Mul stores
 *                      h^sm (fp32, K values per sequence), the down
 *                      projection reads it back with its residual (the
 *                      structure of Alg. 4, which stores h^sm to L3 and loads
 *                      it for the down projection)
 *   FASTTPS_MLP_FUSED  the fused MLP of Section 3.2 with h^sm kept on chip:
 *                      one kernel in which each block computes gate/up and
 *                      siLu_Mul for a slice of the K units, keeps that slice
 *                      in LDS and multiplies it with the matching columns of
 *                      W_down into a partial of y; a second kernel adds the
 *                      blocks' partials in a fixed order with the residual.
 *                      Steps then run the vector projections (the matrix-core
 *                      path is not used), and FASTTPS_DBG_MLP_A has nothing to
 *                      read. Needs W_down in the kernel's slices, which
 *                      fasttps_weights_pack stores (one more copy of W_down)
 *                      only while this path is selected on the layer handle it
 *                      packs with; a step with weights packed otherwise fails
 *                      with FASTTPS_ERR_INVALID_ARG before any launch.
 * Selecting FASTTPS_MLP_FUSED the first time allocates the partial sums
 * (256 x max_batch x D fp32; blocking). Returns FASTTPS_ERR_INVALID_ARG for
 * an unknown path, FASTTPS_ERR_OOM if the allocation fails. */
#define FASTTPS_MLP_SPLIT 0
#define FASTTPS_MLP_FUSED 1
FASTTPS_API int fasttps_set_mlp_path(fasttps_layer* layer, int32_t path);

/* Accuracy-study hook: when enabled, later steps of this layer handle round
 * the softmax weights to bf16 before the PV accumulation, as FlashAttention
 * does with its bf16 P (the softmax row sum stays fp32), so the attention
 * output error of the two can be compared over the context length (the
 * paper's Fig. 8 comparison, Section 4.4, OI and Accuracy). Off by default; a step with it on
 * is not the FastTPS step. */
FASTTPS_API int fasttps_set_attention_p_bf16(fasttps_layer* layer, int32_t enable);

/* Test hook: copy one of the step's fp32 intermediates from the handle's
 * scratch into `dst` (device), on `stream`, after a fasttps_decode_step on the
 * same stream. `which` selects:
 *   FASTTPS_DBG_QKV     [batch, (H + 2 H_kv) d]  q | k | v before RoPE
 *   FASTTPS_DBG_ATTN    [batch, H d]             attention output o
 *   FASTTPS_DBG_H1      [batch, D]               x + W_o o
 *   FASTTPS_DBG_MLP_A   [batch, K]               SiLU(gate) * up (h^sm of Alg. 4)
 *   FASTTPS_DBG_QK_ROPE [batch, (H + H_kv) d]    q | k after the joint RoPE (Alg. 3,
 *                                                Eq. 22), before k is rounded for the cache
 *   FASTTPS_DBG_H       [batch, D]               RMSNorm1(x), the QKV projection's input
 *   FASTTPS_DBG_H2      [batch, D]               RMSNorm2(h1), the gate/up projection's input
 * The last three are written only by steps taken while fasttps_set_debug is
 * on (QK_ROPE by the vector and matrix-core paths, H and H2 by the vector
 * path); reading one the last step did not write fails with
 * FASTTPS_ERR_INVALID_ARG. `bytes` must equal the size of the selected
 * buffer for `batch`. */
#define FASTTPS_DBG_QKV   0
#define FASTTPS_DBG_ATTN  1
#define FASTTPS_DBG_H1    2
#define FASTTPS_DBG_MLP_A 3
#define FASTTPS_DBG_FUSED_WAITS 4  /* int32 [1]: bounded waits of the fused kernel that ran
                                      out since the layer was created (0 when every phase
                                      hand-over completed); `batch` is ignored */
#define FASTTPS_DBG_QK_ROPE 5
#define FASTTPS_DBG_H       6
#define FASTTPS_DBG_H2      7
FASTTPS_API int fasttps_debug_read(fasttps_layer* layer, int32_t which, int32_t batch, void* dst,
                       size_t bytes, void* stream);

/* Test hook: when enabled, later steps of this handle also write the
 * intermediates FASTTPS_DBG_QK_ROPE, FASTTPS_DBG_H and FASTTPS_DBG_H2 (a few
 * KB per sequence, after each kernel's weight or cache stream) into the
 * handle's scratch. Off by default. */
FASTTPS_API int fasttps_set_debug(fasttps_layer* layer, int32_t enable);

/* The argument checks of fasttps_decode_step (cache_elem_bytes 2) or
 * fasttps_decode_step_kv8 (cache_elem_bytes 1) against a layer config,
 * without a handle and without any HIP call: the status a step with these
 * arguments returns before its first launch (handle checks aside).
 *   cfg          host; validated as by fasttps_layer_create
 *   x, k_cache, v_cache, y
 *                only their addresses are examined (null, 16-byte
 *                alignment, overlap); nothing is dereferenced
 *   pos          host, [batch] int32, read
 * Returns FASTTPS_OK, FASTTPS_ERR_INVALID_ARG (null pointer, batch outside
 * [1, max_batch], y overlapping x or a cache, the caches overlapping),
 * FASTTPS_ERR_ALIGNMENT, FASTTPS_ERR_CACHE_FULL (a pos[b] outside
 * [0, N_max)) or a config error. */
FASTTPS_API int fasttps_validate_step(const fasttps_config* cfg, const void* x, const int32_t* pos,
                                      int32_t batch, const void* k_cache, const void* v_cache, const void* y,
                                      int32_t cache_elem_bytes);

/* Measurement hook: time every kernel of the next `max_steps` steps of this
 * handle. Each kernel of those steps is launched with start/stop events that
 * the runtime stamps from the kernel's own dispatch (no extra stream work).
 * fasttps_profile_end waits for the last recorded step, writes the kernel
 * durations in milliseconds to ms[step * FASTTPS_NUM_KERNELS + k] for the
 * n_steps recorded steps (at most max_steps), and releases the events.
 * Kernel k is named by fasttps_kernel_name(k). Steps beyond max_steps run
 * untimed. Not for use under stream capture. */
#define FASTTPS_NUM_KERNELS 7  /* the six kernels of the separate path, then the fused kernel;
                                  a kernel a step does not launch reads 0 (the combine at
                                  batch 1, where the O projection merges the splits and is
                                  timed as kernel 3) */
FASTTPS_API int fasttps_profile_begin(fasttps_layer* layer, int32_t max_steps);
FASTTPS_API int fasttps_profile_end(fasttps_layer* layer, float* ms, int32_t max_steps, int32_t* n_steps);
FASTTPS_API const char* fasttps_kernel_name(int32_t k);

FASTTPS_API int fasttps_weights_free(fasttps_weights* w);
FASTTPS_API int fasttps_layer_destroy(fasttps_layer* layer);

/* Static text of a status code. */
FASTTPS_API const char* fasttps_status_string(int status);
/* Text of the last error on the calling thread ("" if none). */
FASTTPS_API const char* fasttps_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* FASTTPS_H */
