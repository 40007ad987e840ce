/*
 * w4layer.h -- C ABI of the MI355X (gfx950) three-stage W4A16 decoder layer.
 *
 * One Transformer decoder block (RMSNorm, q/k/v projections, RoPE from a
 * precomputed cos/sin table, grouped-query causal attention, o_proj +
 * residual, RMSNorm, SwiGLU MLP + residual; Sec. 3.1, Listings 1-2 of the
 * paper) with 4-bit group-quantised weights and bf16 activations (W4BF16,
 * Sec. 5.1), statically specialised into the paper's three stages
 * (Sec. 4.1, Table 1):
 *
 *   layer_prefill     a whole prompt, no history             (Sec. 4.2)
 *   layer_prefill_kv  a new chunk after a history cache       (Sec. 4.3)
 *   layer_decode      one token per sequence against a cache  (Sec. 4.4)
 *
 * plus the KV-cache calls kv_layout / kv_append (the in-place Concat of
 * Sec. 4.6.3), layer stacks (stack_*), and the model ends around the layers
 * (lm_*: embedding, LM head and greedy sampling of the runtime loop, Sec. 2).
 *
 * Conventions shared by every call
 *   - Return value 0 on success, a negative W4_E* code on failure; the
 *     message of the last failure on the calling thread is layer_last_error().
 *   - Arguments are validated on the host before any HIP call; a call that
 *     fails validation has launched nothing and touched no buffer.
 *   - Pointers documented as "device" are HIP device pointers on the current
 *     device; "host" pointers are ordinary host memory.
 *   - Stage calls are asynchronous on the given stream (a hipStream_t passed
 *     as void*, NULL = default stream), allocate nothing and do not
 *     synchronise.  The caller owns every buffer it passes and must keep it
 *     alive until the stream has drained.
 *   - Device-side values (positions, context lengths) are trusted: an
 *     out-of-range value there is undefined behaviour.
 *
 * Numerics
 *   - Hidden states x and y are fp32 (the block interface of Listing 3 is f32);
 *     the residual stream is never rounded.
 *   - The block's intermediate activations -- the normalised matmul inputs,
 *     q/k after RoPE, v, the attention output and the MLP hidden
 *     activation -- are rounded once to bf16 (round to nearest even), which
 *     is the W4BF16 precision; the K/V cache holds bf16.
 *   - Weights are used exactly: W[k][n] = s[k/G][n] * (q[k][n] - z), sums in
 *     fp32.
 *   - The matrix units take the bf16-rounded activations as fp16 operands.
 *     Every bf16 value of magnitude 2^-17 .. 65280 is an fp16 value, so this
 *     is exact there (below 2^-17 a value moves by less than 3e-8).  A
 *     rounded activation beyond 65504 has no fp16 value: the kernel that
 *     forms it raises W4_FLAG_F16_RANGE in the layer's device error flag
 *     (layer_error) and the call's outputs are not valid.
 */
#ifndef W4LAYER_H
#define W4LAYER_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* ---- error codes --------------------------------------------------------- */
#define W4_OK             0
#define W4_EINVAL        -1  /* null pointer, bad dimension or argument      */
#define W4_EUNSUPPORTED  -2  /* shape or device this library does not handle */
#define W4_ECAPACITY     -3  /* would exceed max_seq or max_batch             */
#define W4_EWORKSPACE    -4  /* workspace missing or smaller than required   */
#define W4_EHIP          -5  /* a HIP runtime call or launch failed          */

/* ---- device error flags (bits; layer_error / lm_error read and clear) ---- */
#define W4_FLAG_WAIT_TIMEOUT 1  /* a wait of the persistent decode timed out: a
                                   block of the launch never got its inputs
                                   (e.g. other work held compute units)      */
#define W4_FLAG_F16_RANGE    2  /* a bf16 activation exceeded 65504 in magnitude
                                   (or was NaN) where an fp16 matrix operand is
                                   formed                                      */
#define W4_FLAG_TOKEN_ID     4  /* lm_embed saw a token id outside the vocabulary */

/* ---- weight formats (layer_config.weight_format) -------------------------
 * The paper compiles W4 group-quantised weights and, besides them, INT8
 * (symmetric or asymmetric) and BF16 weights straight through (Sec. 3.2).
 * All seven linears of a layer share the format.                            */
#define W4_WEIGHTS_INT4 0   /* 4-bit codes, fp16 scales per group of group_size */
#define W4_WEIGHTS_INT8 1   /* 8-bit codes, one fp16 scale (and, asymmetric,
                               one zero point) per output column             */
#define W4_WEIGHTS_BF16 2   /* unquantised bf16 weights                       */

/* ---- types ---------------------------------------------------------------- */

/* Shape of one decoder layer.  Supported: head_dim 64 or 128; n_heads a
 * multiple of n_kv_heads; group_size in {32, 64, 128, 256}; hidden a multiple
 * of 128 and of group_size; n_heads*head_dim a multiple of 128 and of
 * group_size; ffn a multiple of 8; max_seq >= 1; 1 <= max_batch <= 64.
 * rms_eps is added inside the square root of RMSNorm; RoPE uses the
 * rotate-half pairing (i, i + head_dim/2) with angle pos * rope_base^(-2i/d). */
typedef struct layer_config {
    int32_t hidden;
    int32_t n_heads;
    int32_t n_kv_heads;
    int32_t head_dim;
    int32_t ffn;
    int32_t group_size;
    float   rms_eps;
    float   rope_base;
    int32_t max_seq;     /* capacity of the KV cache and of the RoPE table */
    int32_t max_batch;   /* largest decode batch                            */
    int32_t weight_format; /* W4_WEIGHTS_*; 0 (INT4) for zero-initialised
                              configs.  group_size applies to INT4 only.  */
} layer_config;

/* One linear y[M][N] = x[M][K] * W[K][N] in a format that the paper
 * compiles straight through (Sec. 3.2).  All pointers are host pointers,
 * read only during layer_create; the fields a format does not use are
 * ignored.
 * W4_WEIGHTS_INT4 (the canonical GPTQ-style format):
 *   qweight  int32 [K/8][N]: code k = 8r + j of column n in bits 4j..4j+3 of
 *            word [r][n];
 *   scales   fp16 bit patterns [ceil(K/G)][N]: scale of group g = k / G;
 *   zeros    uint8 [ceil(K/G)][N] zero points in 0..15, or NULL for 8;
 *   W[k][n] = scales[k/G][n] * (code - zero).
 * W4_WEIGHTS_INT8 (per output column):
 *   q8       [K][N] codes: with zeros == NULL (symmetric) signed int8 bytes
 *            -128..127 and W[k][n] = scales[n] * q8[k][n]; with zeros
 *            (asymmetric) unsigned bytes 0..255 and
 *            W[k][n] = scales[n] * (q8[k][n] - zeros[n]);
 *   scales   fp16 bit patterns [N];
 *   zeros    uint8 [N] or NULL.
 * W4_WEIGHTS_BF16:
 *   w16      bf16 bit patterns [K][N]; every |W| must be finite and below
 *            4096 (layer_create returns W4_EINVAL otherwise).  Numerics: the
 *            device holds them as fp16 (the matrix cores' operand type of
 *            the layer), which is exact for |W| >= 2^-17 and within 2^-24
 *            below it. */
typedef struct qlinear_host {
    const int32_t*  qweight;
    const uint16_t* scales;
    const uint8_t*  zeros;
    const uint8_t*  q8;
    const uint16_t* w16;
} qlinear_host;

/* All weights of one layer (host pointers).  K x N of each linear, with
 * H = hidden, Q = n_heads*head_dim, V = n_kv_heads*head_dim, F = ffn:
 * q: H x Q, k: H x V, v: H x V, o: Q x H, gate: H x F, up: H x F, down: F x H.
 * attn_norm / mlp_norm: bf16 bit patterns [hidden] (the RMSNorm weights). */
typedef struct layer_weights_host {
    const uint16_t* attn_norm;
    const uint16_t* mlp_norm;
    qlinear_host q, k, v, o, gate, up, down;
} layer_weights_host;

typedef struct layer_s* layer_t;

/* Layout of a K or V cache: bf16 [batch][n_kv_heads][max_seq][head_dim],
 * strides in elements (stride of head_dim is 1), bytes = size of one cache. */
typedef struct kv_desc {
    int32_t batch;
    int32_t n_kv_heads;
    int32_t max_seq;
    int32_t head_dim;
    int64_t stride_b;
    int64_t stride_h;
    int64_t stride_s;
    size_t  bytes;
} kv_desc;

/* ---- lifetime ------------------------------------------------------------ */

/* Validate cfg, repack the host weights into the private device layout,
 * upload them and the fp32 cos/sin table (max_seq x head_dim/2, computed in
 * double precision on the host: the table of Sec. 4.6.2) to the current
 * device.  Synchronous.  On success *out owns all device memory of the layer;
 * no stage call changes it afterwards (scratch state, such as split-K
 * counters, lives in the caller's workspace), so stage calls on different
 * streams may share the handle, each with its own workspace.  One exception:
 * the persistent decode path (layer_set_decode_path; it also serves
 * prefill / prefill_kv calls of a few tokens) needs every compute unit
 * of the device at once, so two of its launches must not overlap on one
 * device; a caller that runs such calls on several streams at once selects
 * path 1.  The diagnostics (profiling, decode stamps) are not for concurrent use.
 * Errors: W4_EINVAL (null), W4_EUNSUPPORTED (shape, or the current device is
 * not gfx950), W4_EHIP (allocation or copy failed). */
int layer_create(const layer_config* cfg, const layer_weights_host* w, layer_t* out);

/* Free the layer's device memory.  The caller must have drained every stream
 * that uses it.  NULL is accepted.  Synchronous. */
int layer_destroy(layer_t layer);

/* The KV-cache layout for a batch of sequences (pure host computation). */
int kv_layout(const layer_config* cfg, int32_t batch, kv_desc* out);

/* Bytes of device workspace a stage call needs: stage 0 prefill (batch 1,
 * T tokens), 1 prefill_kv (batch 1, T tokens, history up to max_ctx), 2
 * decode (batch sequences, context up to max_ctx).  Returns 0 for invalid
 * arguments. */
size_t layer_workspace_size(layer_t layer, int32_t stage, int32_t batch, int32_t T, int32_t max_ctx);

/* ---- the three stages (all device pointers; asynchronous on stream) ---- */

/* Prefill (Sec. 4.2): T >= 1 prompt tokens of one sequence, no history.
 *   x        fp32 [T][hidden] hidden states in;
 *   pos      int32 [T] position_ids (RoPE angles), 0 <= pos < max_seq;
 *   k_cache, v_cache  bf16 [n_kv_heads][max_seq][head_dim] of this sequence
 *            (batch entry of a kv_layout cache); slots 0..T-1 are written,
 *            no other slot is touched;
 *   y        fp32 [T][hidden] out (must not alias x);
 *   ws       workspace of at least layer_workspace_size(layer, 0, 1, T, 0).
 * Errors: W4_EINVAL, W4_ECAPACITY (T > max_seq), W4_EWORKSPACE, W4_EHIP. */
int layer_prefill(layer_t layer, const float* x, const int32_t* pos, int32_t T,
                  void* k_cache, void* v_cache, float* y,
                  void* ws, size_t ws_bytes, void* stream);

/* Prefill_kv (Sec. 4.3): T >= 1 new tokens after hist_len >= 0 cached ones.
 * Reads cache slots 0..hist_len-1, writes slots hist_len..hist_len+T-1, and
 * the new token t attends to slots 0..hist_len+t.  With hist_len = 0 this is
 * exactly layer_prefill.  Other arguments as for layer_prefill; ws of at
 * least layer_workspace_size(layer, 1, 1, T, hist_len).
 * Errors: as layer_prefill, W4_ECAPACITY if hist_len + T > max_seq. */
int layer_prefill_kv(layer_t layer, const float* x, const int32_t* pos, int32_t T, int32_t hist_len,
                     void* k_cache, void* v_cache, float* y,
                     void* ws, size_t ws_bytes, void* stream);

/* Long prompts in segments (the third scenario of Sec. 4.1): tokens
 * 0..chunk-1 by layer_prefill, then every following run of chunk tokens
 * (the last one ragged) by layer_prefill_kv over the tokens before it, all
 * on `stream` in order.  The result equals layer_prefill over the T tokens
 * up to rounding order (each segment's attention sees the cache slots the
 * earlier segments wrote).
 *   x, y     fp32 [T][hidden]; pos int32 [T]; caches as for layer_prefill
 *            (slots 0..T-1 are written);
 *   chunk    tokens per segment, >= 1;
 *   ws       at least layer_prefill_chunked_workspace_size(layer, T, chunk)
 *            bytes, reused by every segment.
 * Errors: as layer_prefill; arguments are validated before the first
 * segment is enqueued. */
size_t layer_prefill_chunked_workspace_size(layer_t layer, int32_t T, int32_t chunk);
int layer_prefill_chunked(layer_t layer, const float* x, const int32_t* pos, int32_t T, int32_t chunk,
                          void* k_cache, void* v_cache, float* y,
                          void* ws, size_t ws_bytes, void* stream);

/* Decode (Sec. 4.4): one new token for each of B sequences.
 *   x         fp32 [B][hidden];
 *   pos       int32 [B] position ids;
 *   ctx_lens  int32 [B] device: cached tokens of sequence b; its new token
 *             is written to slot ctx_lens[b] and attends to slots
 *             0..ctx_lens[b]; every ctx_lens[b] must be <= max_ctx;
 *   max_ctx   host upper bound of ctx_lens, max_ctx + 1 <= max_seq;
 *   attn_mask fp32 [B][max_seq] device, added to the score of slot j (0 to
 *             attend, -inf to mask), or NULL for none; a row whose visible
 *             slots are all -inf produces a zero attention output;
 *   k_cache, v_cache  bf16 caches in the kv_layout(cfg, B) layout;
 *   y         fp32 [B][hidden] out;
 *   ws        at least layer_workspace_size(layer, 2, B, 1, max_ctx).
 * Errors: W4_EINVAL, W4_ECAPACITY (B > max_batch or max_ctx + 1 > max_seq),
 * W4_EUNSUPPORTED (B > 8, or decode path 2 selected and the persistent launch
 * cannot serve the call), W4_EWORKSPACE, W4_EHIP.  Failures the host cannot
 * see (a timed-out wait, an activation beyond the fp16 range) raise bits of
 * the layer's error flag instead: read it with layer_error. */
int layer_decode(layer_t layer, const float* x, const int32_t* pos, const int32_t* ctx_lens,
                 int32_t max_ctx, const float* attn_mask, int32_t B,
                 void* k_cache, void* v_cache, float* y,
                 void* ws, size_t ws_bytes, void* stream);

/* Decode without allocation, for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid
 * it): layer_decode with its workspace taken from a static device array of
 * the library (layer_decode_noalloc_max_bytes() bytes, 32 MiB) instead of a
 * caller buffer.  Each device holds the array from the first layer_create
 * on it until the process ends, and every call on a device shares it, so
 * calls that overlap on one device (other streams, other host threads)
 * race: the caller serialises them.  The call allocates nothing (no
 * hipMalloc, no events: kernel timing does not apply to it); no part of
 * the array has to start at zero.  Arguments as for layer_decode, without
 * ws.  Errors: those of layer_decode; W4_EWORKSPACE if the call needs more
 * scratch than the array holds (the message states both sizes); W4_EHIP if
 * the array was not set up on the layer's device. */
int layer_decode_noalloc(layer_t layer, const float* x, const int32_t* pos, const int32_t* ctx_lens,
                         int32_t max_ctx, const float* attn_mask, int32_t B,
                         void* k_cache, void* v_cache, float* y, void* stream);
size_t layer_decode_noalloc_max_bytes(void);

/* ---- layer stacks (Sec. 4.5, runtime orchestration) ---------------------- */

/* A stack of n_layers layers of one model run back to back on one stream:
 * the output of layer i is the input of layer i + 1.  layers, k_caches and
 * v_caches are host arrays of n_layers entries (each layer has its own
 * caches, in the layouts the single-layer calls take).  x is the input of
 * layer 0 and y receives the output of the last layer (no aliasing); the
 * activations between layers live in the workspace.  All layers must have
 * the same hidden size.  The calls enqueue the layers' kernels and return.
 *
 * stack_workspace_size: bytes for stage 0/1 (prefill / prefill_kv: T tokens,
 * history up to max_ctx) or 2 (decode: batch sequences, context up to
 * max_ctx); 0 for invalid arguments.
 * stack_prefill: every layer runs layer_prefill_kv with hist_len (0: prefill).
 * stack_decode: every layer runs layer_decode with the same pos, ctx_lens,
 * max_ctx, attn_mask and B.
 * Errors: those of the single-layer calls, and W4_EINVAL for a null or
 * mismatched layer list.  Every layer's checks run before the first layer
 * is enqueued, so a failed stack call has launched nothing. */
size_t stack_workspace_size(const layer_t* layers, int32_t n_layers, int32_t stage, int32_t batch,
                            int32_t T, int32_t max_ctx);
int stack_prefill(const layer_t* layers, int32_t n_layers, const float* x, const int32_t* pos,
                  int32_t T, int32_t hist_len, void* const* k_caches, void* const* v_caches,
                  float* y, void* ws, size_t ws_bytes, void* stream);
int stack_decode(const layer_t* layers, int32_t n_layers, const float* x, const int32_t* pos,
                 const int32_t* ctx_lens, int32_t max_ctx, const float* attn_mask, int32_t B,
                 void* const* k_caches, void* const* v_caches, float* y,
                 void* ws, size_t ws_bytes, void* stream);

/* ---- model ends (Sec. 2 inference loop, Sec. 4.5 runtime orchestration) -- */

/* The steps either side of the decoder layers in the runtime loop: the
 * word embedding turns token ids into the first layer's input, the LM head
 * (final RMSNorm + a 4-bit linear hidden x vocab) turns the last layer's
 * output into logits, and greedy sampling picks the next token on the
 * device, so a decode loop needs no host round trip per token.
 * Supported: vocab a positive multiple of 64; hidden a multiple of 128 and
 * of group_size, at most 7680 (the head's GEMV keeps up to 8 whole input
 * rows on chip); group_size in {32, 64, 128, 256}; 1 <= max_batch <= 64.
 * The handle holds only weights, a read-only zero buffer and the embedding
 * error flag: calls on different streams may share it, each lm_head call
 * with its own workspace. */
typedef struct lm_config {
    int32_t vocab;
    int32_t hidden;
    int32_t group_size;
    float   rms_eps;     /* of the final RMSNorm, inside the square root */
    int32_t max_batch;
} lm_config;

/* Host weights, read only during lm_create:
 *   embed       bf16 bit patterns [vocab][hidden]; row t embeds token t;
 *   final_norm  bf16 bit patterns [hidden], the final RMSNorm weight;
 *   head        the LM head, K = hidden, N = vocab, in the qlinear_host
 *               format (codes, fp16 scales, optional zero points). */
typedef struct lm_weights_host {
    const uint16_t* embed;
    const uint16_t* final_norm;
    qlinear_host    head;
} lm_weights_host;

typedef struct lm_s* lm_t;

/* Copies the weights to the current device (the head repacked into the
 * tiled layout of the layer's linears) and returns a handle in *out.
 * Errors: W4_EINVAL (null pointer, non-finite scale), W4_EUNSUPPORTED
 * (shape), W4_EHIP. */
int lm_create(const lm_config* cfg, const lm_weights_host* w, lm_t* out);
int lm_destroy(lm_t lm);

/* Word embedding: x[b][:] = embed[tokens[b]][:] as fp32 (exact), for any
 * number of rows B >= 1 (a whole prompt, or one token per sequence).
 *   tokens  int32 [B] device;  x  fp32 [B][hidden] device out.
 * A token id outside [0, vocab) gives a zero row and sets the handle's
 * error flag (lm_error).  Errors: W4_EINVAL, W4_EHIP. */
int lm_embed(lm_t lm, const int32_t* tokens, int32_t B, float* x, void* stream);

/* Bytes of workspace lm_head needs for B rows; 0 for invalid arguments. */
size_t lm_head_workspace_size(lm_t lm, int32_t B);

/* LM head and greedy sampling:
 *   logits[b][v] = sum_k bf16(RMSNorm(x[b]))[k] * W[k][v]  (fp32 sums, the
 *   normalised row rounded once to bf16 as in the layer), and, when
 *   next_tokens is not NULL, next_tokens[b] = the index of the largest
 *   logit of row b, the lowest index among equal maxima (a NaN logit never
 *   wins; a row of NaNs gives 0).
 *   x            fp32 [B][hidden] device (e.g. the last layer's y);
 *   logits       fp32 [B][vocab] device out;
 *   next_tokens  int32 [B] device out, or NULL;
 *   ws           at least lm_head_workspace_size(lm, B).
 * Deterministic.  Errors: W4_EINVAL, W4_ECAPACITY, W4_EWORKSPACE, W4_EHIP. */
int lm_head(lm_t lm, const float* x, int32_t B, float* logits, int32_t* next_tokens,
            void* ws, size_t ws_bytes, void* stream);

/* Reads and clears the model ends' error flag: *flag holds W4_FLAG_TOKEN_ID
 * if lm_embed saw an id outside the vocabulary, W4_FLAG_F16_RANGE if the
 * final RMSNorm formed an activation beyond the fp16 range, since the last
 * call; 0 if neither.  Waits for the device.  Errors: W4_EINVAL, W4_EHIP. */
int lm_error(lm_t lm, int32_t* flag);

/* One step of the runtime loop's greedy decode (Sec. 2, Sec. 4.5): embed
 * tokens[b] (lm_embed), run every layer's decode on one stream
 * (stack_decode, no attention mask), then the LM head and the greedy pick
 * (lm_head) into logits and next_tokens.  tokens and next_tokens (int32 [B],
 * device) may be the same buffer: the embedding reads it before the pick
 * writes it, in stream order, so a loop feeds each step's picks to the next
 * step without the host.  pos, ctx_lens, max_ctx, caches as for
 * stack_decode; logits fp32 [B][vocab] device out.  ws: at least
 * model_decode_workspace_size(layers, n_layers, lm, B, max_ctx) bytes (0 for
 * invalid arguments).  Every check of every layer (capacity, B <= 8, a
 * forced persistent path that cannot serve the call) runs before the first
 * launch.  If the model ends' error flag or any layer's is set when the pick
 * is done (by this step or an earlier one whose flags were not cleared),
 * every next_tokens[b] is -1, so a loop that stays on the device sees the
 * failure; the next step's embedding then flags the id -1 in turn.
 * Errors: W4_EINVAL, W4_ECAPACITY, W4_EUNSUPPORTED, W4_EWORKSPACE,
 * W4_EHIP. */
size_t model_decode_workspace_size(const layer_t* layers, int32_t n_layers, lm_t lm, int32_t B, int32_t max_ctx);
int model_decode_greedy(const layer_t* layers, int32_t n_layers, lm_t lm, const int32_t* tokens,
                        const int32_t* pos, const int32_t* ctx_lens, int32_t max_ctx, int32_t B,
                        void* const* k_caches, void* const* v_caches, float* logits, int32_t* next_tokens,
                        void* ws, size_t ws_bytes, void* stream);

/* ---- KV cache -------------------------------------------------------------- */

/* In-place Concat (Sec. 4.6.3): copy new keys/values k_new, v_new (bf16
 * [B][T][n_kv_heads][head_dim], device) into cache slots
 * slot_start[b] .. slot_start[b]+T-1 of sequence b (caches in the layout of
 * *desc).  slot_start is a host array [B].  Bit-exact copy; no other slot is
 * touched.  Errors: W4_EINVAL, W4_ECAPACITY (slot range outside the cache or
 * B > desc->batch), W4_EHIP. */
int kv_append(const kv_desc* desc, void* k_cache, void* v_cache,
              const void* k_new, const void* v_new, int32_t B, int32_t T,
              const int32_t* slot_start, void* stream);

/* ---- diagnostics ------------------------------------------------------- */

/* Dequantise linear `which` (0..6 = q, k, v, o, gate, up, down) from the
 * device copy of the weights into out, fp32 [K][N] device, in the order of
 * the canonical format: out[k][n] = s[k/G][n] * (q[k][n] - z) (INT4),
 * s[n] * (q[k][n] - z[n]) (INT8), exact (the product fits fp32); for BF16
 * layers the fp16 value the device holds.  Uses the same unpacking code as
 * the stage kernels.
 * Errors: W4_EINVAL, W4_EHIP. */
int layer_debug_dequant(layer_t layer, int32_t which, float* out, void* stream);

/* Decode implementation (tuning / testing): 0 automatic (default), 1 a
 * sequence of kernels, 2 one persistent launch with one block per CU (B <=
 * 4, INT4 weights without zero points in groups of 64 or more, and the
 * on-chip working set must fit; chosen automatically for B <= 2).  Both compute the same result up to
 * rounding order; the persistent path is deterministic, the kernel sequence
 * adds k-split partials with atomics.  With 2, a decode call the persistent
 * path cannot serve fails with W4_EUNSUPPORTED.  The decode kernels also
 * serve layer_prefill / layer_prefill_kv calls of a few tokens, the tokens
 * as rows of one sequence sharing its cache (row t also attends to the new
 * keys of rows before it): with path 0 up to 2 tokens as the persistent
 * launch and up to 8 as the kernel sequence, with path 2 up to 4 as the
 * persistent launch; path 1 keeps every prefill call on the prefill
 * kernels.  Errors: W4_EINVAL. */
int layer_set_decode_path(layer_t layer, int32_t path);

/* Poll budget of the persistent decode path (testing): the number of polls
 * per thread and launch after which a wait for another block's data gives
 * up, raises W4_FLAG_WAIT_TIMEOUT and lets the launch run to its end (the
 * outputs are then not valid); 0 restores the default (2^20).  A small
 * budget forces the timeout path from the host.  Errors: W4_EINVAL. */
int layer_set_decode_spin_limit(layer_t layer, int32_t polls);

/* Time stamps of the persistent decode path (diagnostics): with on != 0 its
 * launches record per-block wall-clock stamps for layer_decode_phase_times
 * and layer_debug_decode_stamps; off (the default) they record none (the
 * stamp stores lengthen the step).  Errors: W4_EINVAL. */
int layer_set_decode_trace(layer_t layer, int32_t on);

/* Diagnostics of the persistent decode path: durations in microseconds of
 * its five phases in the last completed call (q/k/v, attention with the
 * combine of its chunks, o_proj, gate/up, down), phase p measured from the
 * moment the last block finished phase p-1 (the kernel start for p = 0) to
 * the moment the last block finished phase p (stamps of the last call made
 * with layer_set_decode_trace on), into us_out[5]; and the layer's error
 * flag (W4_FLAG_* bits, not cleared) into *error_flag (nullable).  Waits for
 * the device.  Errors: W4_EINVAL, W4_EHIP. */
int layer_decode_phase_times(layer_t layer, float* us_out, int32_t* error_flag);

/* Raw wall-clock stamps of the last persistent decode call (diagnostics):
 * [0] kernel start (block 0), [1] number of blocks, and at [8 + p*nblocks + j]
 * the time block j passed point p: p = 0..4 the end of the five phases,
 * 5 its start, 23 the end of its prologue, 6/7 the end of the q/k/v RMSNorm /
 * GEMV, 8 q/k/v gathered by its attention unit, 16 RoPE applied, 17 scores
 * done, 18 softmax statistics done, 9 its attention units done, 10 the chunk
 * outputs of its combine slice gathered, 11 the o_proj input gathered, 19
 * o_proj GEMV started, 20/21 its wave / all waves done, 12 h gathered, 22 the
 * MLP RMSNorm done, 13/24 the gate/up GEMV done in wave 0 / all waves, 14 the
 * down input gathered, 15 the down GEMV done (points of work a block does not
 * own keep older values).  Copies min(n, 8 + 32*1024) values.  Waits for the
 * device. */
int layer_debug_decode_stamps(layer_t layer, uint64_t* out, int32_t n);

/* Per-kernel timing for measurement (diagnostics, not for concurrent use).
 * layer_profile_kernel selects, for one stage, the kernel to time (stage 0 and
 * 1, prefill and prefill_kv: 0 rmsnorm, 1 qkv GEMM, 2 attention, 3 o_proj
 * GEMM, 4 rmsnorm, 5 gate/up GEMM, 6 down GEMM; stage 2, decode: 0 qkv GEMV,
 * 1 attention (split + combine), 3 o_proj GEMV, 4 gate/up GEMV, 5 down GEMV,
 * 6 the whole persistent decode launch);
 * kernel < 0 switches timing of that stage off.  While selected, each stage
 * call records a HIP event pair around that launch on the call's stream (at
 * most 4096 pairs per stage until the next read).  Switching timing off and
 * on again with the same kernel keeps the record; selecting another kernel
 * clears it.  layer_profile_read waits for the recorded events of a stage,
 * returns the summed duration in *total_ms and the number of timed launches
 * in *launches, and clears the record.  A layer_prefill_kv call with hist_len 0 counts as stage 0.
 * Errors: W4_EINVAL, W4_EHIP. */
int layer_profile_kernel(layer_t layer, int32_t stage, int32_t kernel);
int layer_profile_read(layer_t layer, int32_t stage, float* total_ms, int32_t* launches);

/* Reads and clears the layer's device error flag: *flag is the OR of the
 * W4_FLAG_* bits raised by its kernels since the last call (0: none).  Waits
 * for the device first (no kernel of the layer is in flight when the flag is
 * read); a call on another host thread that launches meanwhile may have its
 * bits cleared.  Errors: W4_EINVAL, W4_EHIP. */
int layer_error(layer_t layer, int32_t* flag);

/* Ceiling kernels (measurement): what the device sustains on the two
 * resources the stages are bound by (HBM bandwidth for decode, matrix-core
 * throughput for prefill), to report beside the published peaks.
 * w4_ceiling_read streams `bytes` (a multiple of 16, buf 16-byte aligned) of
 * device memory once with 16-byte loads on a grid of `blocks` blocks of 256
 * threads; sink: device memory for blocks * 256 words (a fold of the data).
 * w4_ceiling_mfma runs `iters` (even) iterations of 4 independent fp16 MFMAs on
 * each of 4 waves of `blocks` blocks (big != 0: the GEMM's 32x32x16, else the
 * GEMV's 16x16x32), operands changing every iteration; sink: device memory
 * for blocks * 256 floats; *flop: the floating-point operations of the
 * launch.  Both only enqueue on `stream`.  Errors: W4_EINVAL, W4_EHIP. */
int w4_ceiling_read(const void* buf, size_t bytes, uint32_t* sink, int32_t blocks, void* stream);
int w4_ceiling_mfma(float* sink, int32_t blocks, int32_t iters, int32_t big, double* flop, void* stream);

/* Message of the last failed call on this thread ("" if none). */
const char* layer_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* W4LAYER_H */
