/*
 * keyless.h - C ABI of the keyless-attention library for MI355X (gfx950).
 *
 * Keyless attention scores each query against the cached VALUES through a
 * value-space routing projection instead of separate keys: for one head,
 *     out = softmax(tau * (x W^Q W^R) (X W^V)^T) (X W^V),   tau = 1/sqrt(d_head)
 * (Eq. 2; the per-pair score is Eq. 4). Decoding therefore needs only a
 * value-only cache (Section 3): o = sum_i alpha_i v_i with
 * alpha_i proportional to exp(tau <q~, v_i>) over every cached row, the current
 * token's value included.
 *
 * Conventions for every call below:
 *  - All tensor arguments are DEVICE pointers to row-major, contiguous memory
 *    owned by the caller. The library never allocates, frees or synchronises
 *    inside these calls; every kernel is enqueued on `stream` (a hipStream_t;
 *    NULL means the default stream) and the call returns without waiting.
 *  - Weights right-multiply activations, as in the paper's X W.
 *  - Grouped heads (Section 3, GQA): query head h reads value group
 *    g = h / (H / G); H must be a multiple of G. G = H is multi-head, G = 1 is
 *    multi-query.
 *  - Errors: host-side validation returns a negative kl_status and sets a
 *    thread-local message readable with keyless_last_error(). Nothing is
 *    enqueued when validation fails. KL_ERR_HIP reports a failed launch.
 *  - Device-resident integers (lengths, block tables) are not validated on
 *    the host (that would need a synchronisation). The kernels clamp a length
 *    to [0, capacity], treat block ids outside [0, num_blocks) as empty rows,
 *    and drop appended rows that fall beyond capacity, so bad device data can
 *    give wrong results but never an out-of-bounds access.
 *  - Supported: d_head in {64, 128}; H / G any value for prefill, 1 to 8 for
 *    decode (also 16 or 32 for a bf16 cache with d_head 128); element type bf16
 *    (stored as raw 16-bit words) or fp32; arithmetic is fp32 in both cases.
 */
#ifndef KEYLESS_H_
#define KEYLESS_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  KL_OK = 0,
  KL_ERR_INVALID_ARG = -1,  /* null pointer, bad size, inconsistent shapes      */
  KL_ERR_UNSUPPORTED = -2,  /* valid request this build does not implement      */
  KL_ERR_WORKSPACE = -3,    /* workspace missing or smaller than required       */
  KL_ERR_HIP = -4           /* a HIP runtime call or kernel launch failed       */
} kl_status;

typedef enum { KL_F32 = 0, KL_BF16 = 1 } kl_dtype;

typedef enum { KL_CONTIGUOUS = 0, KL_PAGED = 1 } kl_layout;

/*
 * Value-only cache descriptor (Section 3: each head or group keeps its own
 * rows v_i in R^{d_head}). The descriptor itself lives in host memory; `data`
 * and `block_table` are device pointers owned by the caller.
 *
 *  KL_CONTIGUOUS: data is [B, G, L_max, d_head]; row i of sequence b, group g
 *                 is data[b][g][i]. Capacity per sequence = L_max.
 *  KL_PAGED:      data is [num_blocks, G, block_size, d_head]; row i of
 *                 sequence b lives in block block_table[b * max_blocks_per_seq
 *                 + i / block_size] at slot i % block_size. block_size must be
 *                 a power of two and a multiple of 16. Capacity per sequence =
 *                 max_blocks_per_seq * block_size.
 */
typedef struct {
  void* data;
  kl_dtype dtype;
  kl_layout layout;
  int G;
  int d_head;
  int L_max;                  /* contiguous only                                */
  int block_size;             /* paged only                                     */
  int num_blocks;             /* paged only                                     */
  int max_blocks_per_seq;     /* paged only                                     */
  const int32_t* block_table; /* paged only: [B, max_blocks_per_seq], device    */
} kl_value_cache;

/*
 * keyless_latent_decode - one decode step over a latent value-only cache
 * (Section 3, Eq. 15). The cache holds V* = X W^V_pre (rank r rows) instead of
 * the values; each query head h expands them with its own W^V_{h,post}:
 *   q*[b,h]  = q_routed[b,h] W_post[h]^T                 (absorbed query, r wide)
 *   o*[b,h]  = sum_{i < lengths[b]} alpha_i V*_i,  alpha = softmax_i(scale <q*, V*_i>)
 *   out[b,h] = o*[b,h] W_post[h]
 * over latent group g = h / (H / G) of the cache.
 *   q_routed      [B, H, d_head], the routed queries q~ (cache dtype)
 *   W_post        [H, r, d_head]: W^V_{h,post} per query head (a shared or per-group
 *                 expansion is passed repeated), cache dtype
 *   latent_cache  descriptor as for keyless_decode with d_head = r (64 or 128) and
 *                 G latent groups (G = 1: one latent shared by all heads)
 *   lengths       [B] int32 on the device, clamped to [0, capacity]
 *   d_head        64 or 128
 *   scale         >= 0; 0 selects 1/sqrt(r) as in Eq. 15
 *   out           [B, H, d_head]
 *   ws, ws_bytes  keyless_latent_decode_workspace_size(...) bytes, 16-byte aligned:
 *                 q* and o* (B*H*r elements each, rounded up to 256 bytes) and the
 *                 decode's own workspace
 * q_routed and W_post 16-byte aligned. H/G as for keyless_decode (16 or 32 only
 * for bf16 with r = 128). q* and o* are
 * rounded to the cache dtype; fp32 accumulation throughout. An empty cache gives
 * a zero row. Errors: KL_ERR_* before any launch.
 */
int keyless_latent_decode(const void* q_routed, const void* W_post,
                          const kl_value_cache* latent_cache, const int32_t* lengths, int B, int H,
                          int d_head, float scale, void* out, void* ws, size_t ws_bytes,
                          void* stream);
size_t keyless_latent_decode_workspace_size(const kl_value_cache* latent_cache, int B, int H,
                                            int d_head);

/*
 * keyless_fold_routing - folded query weight W~^Q_h = W^Q_h W^R_h for every
 * head h (Section 2.1: the two query matrices are composed once before
 * inference; Section 5.5 uses the fused matrix for decoding).
 *   W_Q   [d_model, H * d_head]   head h owns columns h*d_head .. h*d_head+d_head-1
 *   W_R   [H, d_head, d_head]     one routing matrix per query head
 *   Wt_Q  [d_model, H * d_head]   output, same dtype
 * fp32 accumulation; a bf16 result is rounded to nearest even once.
 */
int keyless_fold_routing(const void* W_Q, const void* W_R, int d_model, int H, int d_head,
                         kl_dtype dtype, void* Wt_Q, void* stream);

/*
 * keyless_prefill - keyless self-attention over N tokens (Eq. 2 with the
 * score of Eq. 4; Section 3 multi-head/grouped forms).
 *   x       [B, N, d_model]
 *   W_Q     [d_model, H * d_head]; if W_R is NULL it is taken as the folded W~^Q
 *   W_R     [H, d_head, d_head] or NULL
 *   W_V     [d_model, G * d_head]
 *   causal  nonzero: token i attends to tokens j <= i (itself included)
 *   scale   softmax temperature, >= 0; 0 selects 1/sqrt(d_head)
 *   out     [B, N, H, d_head]
 *   q_routed_out  [B, N, H, d_head] or NULL (the routed queries x W~^Q)
 *   v_out         [B, N, G, d_head] or NULL (the values to append to the cache)
 *   ws, ws_bytes  workspace of at least keyless_prefill_workspace_size(...) bytes
 * There is no key projection. bf16 uses MFMA with fp32 accumulation; the
 * routed queries and values are rounded to bf16 once, as they would be cached.
 * For bf16 the weights are folded and packed into the workspace on every call
 * (d_model must be a multiple of 64; x, the weights, out, q_routed_out, v_out
 * and ws 16-byte aligned, else KL_ERR_INVALID_ARG before any launch); callers
 * that keep weights resident should pack once with keyless_pack_weights and
 * call keyless_prefill_packed.
 */
int keyless_prefill(const void* x, const void* W_Q, const void* W_R, const void* W_V, int B,
                    int N, int d_model, int H, int G, int d_head, int causal, float scale,
                    kl_dtype dtype, void* out, void* q_routed_out, void* v_out, void* ws,
                    size_t ws_bytes, void* stream);

size_t keyless_prefill_workspace_size(int B, int N, int d_model, int H, int G, int d_head,
                                      kl_dtype dtype, int has_W_R, int has_q_routed_out,
                                      int has_v_out);

/*
 * keyless_pack_weights - the one-time weight preparation before inference
 * (Section 2.1: W^Q and W^R are composed into W~^Q once; Section 5.5 does the
 * same before decoding). Writes, for the bf16 path, the packed matrix
 *   packed [(H + G) * d_head, d_model]:  row n < H*d_head is column n of
 *   W~^Q = W^Q W^R (per head; W^Q itself when W_R is NULL), row H*d_head + n
 *   is column n of W^V,
 * i.e. the projection weights transposed so that d_model is contiguous, the
 * layout the MFMA projection reads. fp32 accumulation for the fold (a matrix
 * core product per head), one rounding to bf16; the W^V rows (and the W^Q rows
 * when W_R is NULL) are copied bit for bit. packed holds
 * keyless_packed_weights_size(...) bytes. bf16 and d_head 64 or 128 only
 * (KL_ERR_UNSUPPORTED otherwise); every pointer 16-byte aligned
 * (KL_ERR_INVALID_ARG otherwise).
 */
size_t keyless_packed_weights_size(int d_model, int H, int G, int d_head, kl_dtype dtype);
int keyless_pack_weights(const void* W_Q, const void* W_R, const void* W_V, int d_model, int H,
                         int G, int d_head, kl_dtype dtype, void* packed, void* stream);

/*
 * keyless_prefill_packed - keyless_prefill with weights prepared by
 * keyless_pack_weights (bf16 only; d_model a multiple of 64; every pointer
 * 16-byte aligned, else KL_ERR_INVALID_ARG before any launch). The workspace is
 * needed only for q_routed / v when those outputs are NULL:
 * B*N*H*d_head*2 and B*N*G*d_head*2 bytes, each rounded up to 256.
 */
int keyless_prefill_packed(const void* x, const void* packed, int B, int N, int d_model, int H,
                           int G, int d_head, int causal, float scale, kl_dtype dtype, void* out,
                           void* q_routed_out, void* v_out, void* ws, size_t ws_bytes,
                           void* stream);

/*
 * keyless_cross_attention - keyless cross-attention (Section 2.5, Eq. 14): the
 * queries come from one sequence, the values, which also route, from another:
 *   out[b, i, h] = softmax_j(scale <q~_i, v_j>) summed against v_j, where
 *   q~_i = xa[b, i] W~^Q_h (i < N_a) and v_j = xb[b, j] W^V_g (j < N_b),
 *   g = h / (H / G); every query sees every value (no mask).
 *   xa      [B, N_a, d_model]   the attending sequence (e.g. the decoder side)
 *   xb      [B, N_b, d_model]   the attended sequence (e.g. an encoder or
 *                               another modality); N_a and N_b are independent;
 *                               NULL is accepted when N_b = 0
 *   W_Q, W_R, W_V, scale, dtype as for keyless_prefill
 *   out     [B, N_a, H, d_head]
 *   q_routed_out  [B, N_a, H, d_head] or NULL
 *   v_out         [B, N_b, G, d_head] or NULL (the values, cacheable once per xb)
 *   ws, ws_bytes  workspace of at least keyless_cross_attention_workspace_size(...)
 * N_b = 0 gives zero output rows (nothing to average). xa == xb with N_a == N_b
 * is keyless_prefill with causal = 0. Same precision and errors as
 * keyless_prefill.
 */
int keyless_cross_attention(const void* xa, const void* xb, const void* W_Q, const void* W_R,
                            const void* W_V, int B, int N_a, int N_b, int d_model, int H, int G,
                            int d_head, float scale, kl_dtype dtype, void* out,
                            void* q_routed_out, void* v_out, void* ws, size_t ws_bytes,
                            void* stream);

size_t keyless_cross_attention_workspace_size(int B, int N_a, int N_b, int d_model, int H, int G,
                                              int d_head, kl_dtype dtype, int has_W_R,
                                              int has_q_routed_out, int has_v_out);

/*
 * keyless_cross_attention_packed - keyless_cross_attention with weights prepared
 * by keyless_pack_weights (bf16 only; d_model a multiple of 64): the routed
 * queries come from the first H*d_head packed rows applied to xa, the values
 * from the remaining G*d_head rows applied to xb. The workspace is needed only
 * for q_routed / v when those outputs are NULL: B*N_a*H*d_head*2 and
 * B*N_b*G*d_head*2 bytes, each rounded up to 256.
 */
int keyless_cross_attention_packed(const void* xa, const void* xb, const void* packed, int B,
                                   int N_a, int N_b, int d_model, int H, int G, int d_head,
                                   float scale, kl_dtype dtype, void* out, void* q_routed_out,
                                   void* v_out, void* ws, size_t ws_bytes, void* stream);

/*
 * keyless_attention_forward - the attention of Eq. 2 (score Eq. 4) on routed
 * queries and values already projected, also writing each row's log-sum-exp for
 * the backward pass:
 *   q_routed [B, N, H, d_head], v [B, N, G, d_head], out [B, N, H, d_head], all
 *   contiguous and 16-byte aligned, in `dtype`
 *   lse      [B, H, N] fp32, or NULL: ln sum_j exp(scale <q~_i, v_j>) over the
 *            rows j that row i sees
 *   out_f32  [B, N, H, d_head] fp32, or NULL: the output before its rounding to
 *            `dtype` (for keyless_attention_backward), 16-byte aligned
 * causal, scale, precision and errors as for keyless_prefill.
 */
int keyless_attention_forward(const void* q_routed, const void* v, int B, int N, int H, int G,
                              int d_head, int causal, float scale, kl_dtype dtype, void* out,
                              float* lse, float* out_f32, void* stream);

/*
 * keyless_attention_backward - gradients of the keyless attention (Section 2.3)
 * with respect to the routed queries and the values, given dL/dO:
 *   dS  = P * (dO V^T - rowsum(dO * O)),  P the forward's weights (from lse)
 *   dq_routed = scale dS V
 *   dv        = P^T dO + scale dS^T Q~   (the retrieval and routing terms of
 *               Eq. 6; a value group sums them over its H/G heads)
 *   q_routed, v, out (the forward's output), dout [B, N, H, d_head] and lse as
 *   written by keyless_attention_forward with the same causal and scale;
 *   out_f32 the forward's fp32 output, or NULL. The row sums rowsum(P * dP) =
 *   rowsum(dO * O) are taken from out_f32 when given; otherwise, for bf16, from P
 *   and dP in an extra sweep over the values (rowsum(dO * O) over the bf16
 *   output would carry its rounding into every dP - rowsum);
 *   dq_routed [B, N, H, d_head], dv [B, N, G, d_head]; all 16-byte aligned.
 *   ws, ws_bytes  keyless_attention_backward_workspace_size(B, N, H) bytes (the
 *                 per-row rowsum(dO * O), B*H*N floats)
 * Self-attention only (the value rows are the query rows). bf16 with d_head 64
 * or 128 runs on MFMA (P and dS rounded to bf16 for the products, fp32
 * accumulation); fp32 on the vector ALU. Every output element is written once
 * (no atomics): results are deterministic.
 */
int keyless_attention_backward(const void* q_routed, const void* v, const void* out,
                               const float* out_f32, const void* dout, const float* lse, int B,
                               int N, int H, int G,
                               int d_head, int causal, float scale, kl_dtype dtype, void* dq_routed,
                               void* dv, void* ws, size_t ws_bytes, void* stream);
size_t keyless_attention_backward_workspace_size(int B, int N, int H);

/*
 * keyless_weight_gradients - the rest of the backward pass through the
 * projections Q_h = X W^Q_h, Q~_h = Q_h W^R_h, V = X W^V (Section 2.3):
 *   dW_R[h] = (X W^Q_h)^T dq_routed_h           (Eq. 5)
 *   dQ_h    = dq_routed_h W_R[h]^T
 *   dW_Q    = X^T dQ,   dW_V = X^T dv           (Eq. 6; dv holds both terms)
 *   dx      = dQ W_Q^T + dv W_V^T
 * summed over the batch. x [B, N, d_model]; W_Q [d_model, H*d_head], W_R [H,
 * d_head, d_head], W_V [d_model, G*d_head]; dq_routed, dv as written by
 * keyless_attention_backward. Outputs dW_Q, dW_R, dW_V (the weights' shapes) and
 * dx [B, N, d_model]; any of them may be NULL to skip it. ws, ws_bytes:
 * keyless_weight_gradients_workspace_size(...) bytes, 16-byte aligned.
 * bf16 with 16-byte aligned inputs and workspace, and d_head and d_model
 * multiples of 64, runs every product above on the matrix cores (fp32
 * accumulation; X W^Q and dQ rounded to bf16 once, as stored intermediates);
 * other cases run the same products on the generic fp32-arithmetic kernel.
 * Returns KL_ERR_WORKSPACE when the workspace is too small.
 */
int keyless_weight_gradients(const void* x, const void* W_Q, const void* W_R, const void* W_V,
                             const void* dq_routed, const void* dv, int B, int N, int d_model,
                             int H, int G, int d_head, kl_dtype dtype, void* dW_Q, void* dW_R,
                             void* dW_V, void* dx, void* ws, size_t ws_bytes, void* stream);
size_t keyless_weight_gradients_workspace_size(int B, int N, int d_model, int H, int G,
                                               int d_head, kl_dtype dtype);

/*
 * keyless_decode_project - the projections of one decode step (Section 3: the
 * current token's routed query q~_{n+1} and its value v_{n+1}, i.e. the
 * projections of Eq. 2 for one token per sequence), from weights prepared by
 * keyless_pack_weights:
 *   q~[b, h] = x[b] W~^Q_h      v[b, g] = x[b] W^V_g
 *   x              [B, d_model] bf16, the current tokens
 *   packed         [(H + G) * d_head, d_model] bf16 (keyless_pack_weights)
 *   q_routed_out   [B, H, d_head] bf16
 *   v_out          [B, G, d_head] bf16, or NULL
 *   cache          bf16 value cache with G groups of d_head, or NULL: when given,
 *                  v[b] is also written at position lengths_before[b] of sequence b
 *                  (value_cache_append with T = 1, same dropping rules), so the
 *                  decode that follows (with lengths_before[b] + 1) reads it
 *   lengths_before [B] int32 on the device; required with a cache
 * bf16 only; d_model a multiple of 32 and at most 16384; x and packed 16-byte
 * aligned. fp32 accumulation, one rounding to bf16 (the cached value and v_out are
 * the same bits). Bound by the weight bytes: each packed row is read once per 16
 * sequences. Errors: KL_ERR_INVALID_ARG / KL_ERR_UNSUPPORTED before any launch.
 */
int keyless_decode_project(const void* x, const void* packed, int B, int d_model, int H, int G,
                           int d_head, kl_dtype dtype, void* q_routed_out, void* v_out,
                           const kl_value_cache* cache, const int32_t* lengths_before,
                           void* stream);

/*
 * keyless_decode - one decode step over a value-only cache (Section 3):
 *   out[b,h] = sum_{i < lengths[b]} alpha_i v_i,
 *   alpha_i = exp(scale <q_routed[b,h], v_i>) / sum_j exp(scale <q_routed[b,h], v_j>)
 * with v_i the rows of group h / (H / G) of sequence b. H / G is 1 to 8, and
 * also 16 or 32 for a bf16 cache with d_head 128 (KL_ERR_UNSUPPORTED otherwise).
 *   q_routed [B, H, d_head]  routed queries x W~^Q of the current tokens (cache dtype)
 *   cache    value-only cache descriptor (host pointer)
 *   lengths  [B] int32, device: rows per sequence, the current token's value
 *            included (append it first with value_cache_append)
 *   scale    0 selects 1/sqrt(d_head) (lambda = 1 in the Section 3 weight)
 *   out      [B, H, d_head], cache dtype. lengths[b] == 0 gives a zero row.
 *   ws       at least keyless_decode_workspace_size(...) bytes (may be 0, then
 *            ws may be NULL). Calls that run at the same time must not share it.
 * Each cached value tile is read from HBM once and used both for the scores
 * and for the weighted sum. Work split (the built-in choice): a contiguous
 * cache with at least 256 (b, group) pairs gets one workgroup per pair and no
 * merge; otherwise a fixed set of 512 workgroups shares the 16-row tiles of
 * all pairs evenly (a plan kernel prefix-sums the lengths on the device), and
 * a merge kernel combines the pairs that several workgroups shared, always in
 * the same order, so results are reproducible for fixed inputs. The workspace
 * contents need not be initialised and are not preserved.
 */
int keyless_decode(const void* q_routed, const kl_value_cache* cache, const int32_t* lengths,
                   int B, int H, float scale, void* out, void* ws, size_t ws_bytes, void* stream);

/*
 * keyless_decode_append - one whole decode step over the value-only cache
 * (Section 3: the step's value v_{n+1} joins the cache and the step's query
 * attends over all n+1 values) in one launch: the same result as
 * value_cache_append(cache, v_new, lengths_before) followed by keyless_decode
 * over lengths_before[b] + 1 rows, with the new row taken from v_new rather
 * than read back from the cache.
 *   v_new           [B, G, d_head], cache dtype, 16-byte aligned
 *   lengths_before  [B] int32 on the device: rows already cached; the new row goes
 *                   to position lengths_before[b] (dropped past the capacity or a
 *                   block outside the cache, as value_cache_append drops it)
 * Other arguments, workspace and errors as for keyless_decode (which uses the
 * same work split for lengths_before + 1 rows).
 */
int keyless_decode_append(const void* q_routed, const void* v_new, const kl_value_cache* cache,
                          const int32_t* lengths_before, int B, int H, float scale, void* out,
                          void* ws, size_t ws_bytes, void* stream);

/*
 * keyless_decode_noalloc - keyless_decode for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, harnesses
 * that forbid allocation): the same result, kernels and work split, with the
 * workspace taken from a fixed scratch array of 16 MiB that the library holds
 * on each GPU it runs on (resolved once per device, kept until the process
 * ends). The caller passes only inputs and outputs; nothing is allocated,
 * freed or synchronised. A decode whose workspace
 * (keyless_decode_workspace_size with chunk_rows 0) exceeds 16 MiB returns
 * KL_ERR_UNSUPPORTED before any launch. All calls on one GPU share its scratch
 * array, so calls that overlap on one GPU (other streams, other host threads)
 * race and must be ordered by the caller; the scratch needs no clearing, as
 * every call writes each workspace entry before reading it. Other arguments and
 * errors as for keyless_decode.
 */
int keyless_decode_noalloc(const void* q_routed, const kl_value_cache* cache,
                           const int32_t* lengths, int B, int H, float scale, void* out,
                           void* stream);

/* As keyless_decode, with the cache length split into chunks of chunk_rows
 * rows fixed by the caller (a multiple of 64; 0 selects the built-in choice):
 * one workgroup per (b, group, chunk), then a merge of the chunks of each
 * (b, h) in chunk order. A chunk at least as long as the capacity gives one
 * split and no merge kernel. At most 1024 splits per sequence. */
int keyless_decode_chunked(const void* q_routed, const kl_value_cache* cache,
                           const int32_t* lengths, int B, int H, float scale, void* out,
                           void* ws, size_t ws_bytes, int chunk_rows, void* stream);

/* Workspace bytes for keyless_decode_chunked / standard_decode_chunked with
 * these arguments (chunk_rows 0 for keyless_decode / standard_decode): fp32
 * partial rows (d_head + 2 floats per head and split) plus, in the shared-tile
 * mode, a plan of B + 3 ints; 0 when no merge is needed. Host-only; depends on
 * the descriptor's layout and capacity, not on the lengths. */
size_t keyless_decode_workspace_size(const kl_value_cache* cache, int B, int H, int chunk_rows);

/*
 * value_cache_append - write T new value rows per sequence into the cache
 * (Section 3: the new value v_{n+1} joins the cache before the decode step
 * that reads it).
 *   values          [B, T, G, d_head], cache dtype
 *   lengths_before  [B] int32, device: rows already cached; row t of sequence
 *                   b goes to position lengths_before[b] + t
 * Positions at or beyond the capacity are dropped. `lengths` is not updated:
 * the caller owns it.
 */
int value_cache_append(const kl_value_cache* cache, const void* values,
                       const int32_t* lengths_before, int B, int T, void* stream);

/*
 * standard_decode - the comparison baseline: standard attention of Eq. 1 for
 * one new query per sequence over a key cache and a value cache with the same
 * layout as `v_cache` (scores <q, k_i>, weights applied to v_i). Same tiling,
 * split and merge as keyless_decode; it reads twice the bytes.
 */
int standard_decode(const void* q, const kl_value_cache* k_cache, const kl_value_cache* v_cache,
                    const int32_t* lengths, int B, int H, float scale, void* out, void* ws,
                    size_t ws_bytes, void* stream);

int standard_decode_chunked(const void* q, const kl_value_cache* k_cache,
                            const kl_value_cache* v_cache, const int32_t* lengths, int B, int H,
                            float scale, void* out, void* ws, size_t ws_bytes, int chunk_rows,
                            void* stream);

/*
 * keyless_set_kernel_timer - instrumentation for benchmarks. When both handles
 * are non-NULL (hipEvent_t created by the caller), every later decode or
 * standard_decode call made on this thread records `start` on its stream just
 * before its split kernel (the kernel that reads the cache) and `stop` just
 * after it, so that kernel can be timed alone. NULL, NULL turns it off.
 */
void keyless_set_kernel_timer(void* start_event, void* stop_event);

/*
 * keyless_probe_read, keyless_probe_mfma - instrumentation for benchmarks: the
 * practical ceilings that the roofline fractions of the kernels above are read
 * against. Neither computes anything of the method.
 *
 * keyless_probe_read reads the `bytes` bytes at device pointer `src` once
 * (16-byte non-temporal loads; each of `workgroups` workgroups of 256 lanes
 * streams a contiguous share) and writes nothing but, in a case no real input
 * is expected to give, one word to the device word `sink`. `src` must be 16-byte aligned and `bytes`
 * a multiple of 16; `workgroups` in [1, 2^20]. Enqueued on `stream`.
 *
 * keyless_probe_mfma runs, in each of `workgroups` workgroups of 4 waves,
 * `iters` rounds of 16 independent bf16 matrix-core products of 16 x 16 x 32
 * (workgroups x 4 x iters x 16 x 16384 FLOP in all) on constant operands, and
 * likewise writes at most one word to the device float `sink`. `iters` >= 1,
 * `workgroups` in [1, 2^20].
 *
 * Both return KL_ERR_INVALID_ARG for arguments outside these ranges.
 */
int keyless_probe_read(const void* src, size_t bytes, unsigned* sink, int workgroups,
                       void* stream);
int keyless_probe_mfma(float* sink, int iters, int workgroups, void* stream);

/* Thread-local text describing the last non-OK status returned on this thread. */
const char* keyless_last_error(void);

/* Library version string. */
const char* keyless_version(void);

#ifdef __cplusplus
}
#endif

#endif /* KEYLESS_H_ */
