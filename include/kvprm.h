/*
 * kvprm.h - C ABI of the KV-PRM verify-token scoring library for AMD Instinct MI355X (gfx950).
 *
 * KV-PRM (section 4.1, Eq. (score)) scores a candidate trajectory by pushing one appended
 * "verify" token through the adapter-merged decoder f_{theta+dtheta}, conditioned on the key/
 * value cache the generator already produced for that trajectory, and reading two judgment
 * logits: P(+) = softmax([z_-, z_+]) at the "+" entry = sigmoid(z_+ - z_-). The cost is one
 * query against L cached positions per layer (Eq. (cost_kv)), O(d L) instead of the O(d L^2)
 * re-encode of the text (Eq. (1)).
 *
 * Conventions for every entry point
 *   - All tensor pointers are DEVICE pointers unless the name ends in _host. The caller owns
 *     every buffer; the library never frees, never writes the cache (except kvprm_steer, which
 *     exists to update it), the page table or the weights, and never allocates device memory
 *     in any call (the caller passes a workspace sized by the matching kvprm_workspace_size*
 *     query), so every scoring call can be captured in a HIP graph (no memset nodes either;
 *     not in the KVPRM_DEBUG mode below, which synchronises).
 *   - Calls only enqueue work on `stream` (a hipStream_t; NULL = the null stream) and never
 *     synchronise the host. Outputs are valid once the stream reaches that point.
 *   - Arguments are validated on the host before anything is enqueued; on any error nothing
 *     is enqueued. The returned status says what failed; kvprm_last_error() has the text.
 *   - A handle is immutable after kvprm_create. Concurrent calls on one handle are safe when
 *     they use distinct workspaces and outputs.
 *   - Out-of-range physical page ids in the page table are undefined behaviour: the kernels do
 *     not check them. With the environment variable KVPRM_DEBUG=1 set when the handle is
 *     created, the calls that read the cache copy lengths and page table to the host (on
 *     `stream`, then synchronising it) and return KVPRM_E_INVALID, before enqueueing anything,
 *     for any page id outside [0, num_pages) among the pages a candidate reads, for a
 *     lengths_host entry that differs from the device length, and (kvprm_score_grad,
 *     kvprm_steer) for a physical page read by two candidates.
 *
 * Model structure (the paper names only "decoder-only transformer"; the block follows the
 * Qwen3/Llama family it evaluates): pre-norm RMSNorm -> Q/K/V projections -> rotate-half
 * rotary embedding at the verify position -> grouped-query attention (q-head h reads kv-head
 * floor(h / g), g = n_q / n_kv) -> output projection -> residual; RMSNorm -> SwiGLU FFN ->
 * residual; final RMSNorm -> reward vector. No biases. Matrices are [out, in] (layout: see
 * kvprm_layer_weights).
 */
#ifndef KVPRM_H
#define KVPRM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct kvprm_handle_s *kvprm_handle;

typedef enum {
  KVPRM_OK = 0,
  KVPRM_E_INVALID = 1,     /* a null pointer, a negative size, inconsistent arguments */
  KVPRM_E_UNSUPPORTED = 2, /* a valid configuration this build does not implement */
  KVPRM_E_WORKSPACE = 3,   /* workspace pointer null or smaller than kvprm_workspace_size */
  KVPRM_E_HIP = 4,         /* a HIP runtime call or kernel launch failed */
  KVPRM_E_INTERNAL = 5
} kvprm_status;

typedef enum { KVPRM_F32 = 0, KVPRM_BF16 = 1, KVPRM_FP8_E4M3 = 2 } kvprm_dtype;

/* Model shape. Supported: head_dim in {64, 128}; page_size == 16; num_q_heads a multiple of
 * num_kv_heads; weight_dtype F32 with kv_dtype F32, or weight_dtype BF16 with kv_dtype BF16 or
 * FP8_E4M3 (OCP E4M3FN: bias 7, max 448, no infinities). */
typedef struct {
  int32_t num_layers;   /* N_L */
  int32_t hidden;       /* H, a multiple of 64 */
  int32_t num_q_heads;  /* n_q */
  int32_t num_kv_heads; /* n_kv */
  int32_t head_dim;     /* d_h */
  int32_t ffn_dim;      /* F, a multiple of 64 */
  float rope_theta;     /* rotary base theta; angle of pair i at position p is p * theta^(-2i/d_h) */
  float rms_eps;        /* RMSNorm epsilon: y = x / sqrt(mean(x^2) + eps) * gamma */
  kvprm_dtype weight_dtype;
  kvprm_dtype kv_dtype;
  int32_t page_size; /* tokens per cache page; must be 16 */
} kvprm_model_desc;

/* One decoder layer of the readout weights theta + dtheta (for kvprm_score the LoRA update is
 * merged into the base weights by the caller: W' = W + (alpha / r) B A; section 4.1 and the
 * hyperparameter table; kvprm_score_lora takes the base weights and the factors instead).
 * Element type weight_dtype. Matrices are [out, in]: row-major for F32 weights; for BF16
 * weights in the packed tile layout written by kvprm_pack_weight (so that the matrix cores
 * stream them contiguously). Gains are plain vectors. */
typedef struct {
  const void *attn_norm; /* [H]                gain of the attention RMSNorm */
  const void *wq;        /* [n_q * d_h, H]     head h occupies rows [h d_h, (h+1) d_h) */
  const void *wk;        /* [n_kv * d_h, H] */
  const void *wv;        /* [n_kv * d_h, H] */
  const void *wo;        /* [H, n_q * d_h] */
  const void *ffn_norm;  /* [H]                gain of the FFN RMSNorm */
  const void *w_gate;    /* [F, H] */
  const void *w_up;      /* [F, H] */
  const void *w_down;    /* [H, F] */
} kvprm_layer_weights;

typedef struct {
  const kvprm_layer_weights *layers; /* HOST array [num_layers] of device pointers */
  const void *verify_embed;          /* [H] embedding row of the verify token (weight_dtype) */
  const void *final_norm;            /* [H] gain of the final RMSNorm (weight_dtype) */
  const void *reward_w;              /* [H] W_out[+] - W_out[-] (weight_dtype) */
  float reward_b;                    /* b[+] - b[-] */
} kvprm_readout_weights;

/* Paged KV cache written by the generator (adapter off; section 4.1). Keys are stored after
 * the rotary embedding of their own position; values are not rotated.
 *   pool layout: [num_layers][num_pages][num_kv_heads][tile]
 *   x = 16 bytes / element size (4 fp32, 8 bf16, 16 fp8), r = x / 4
 *   K tile (page_size x d_h values): [d_h / x][page_size][x]: element (slot s, dim m) at
 *            ((m / x) * 16 + s) * x + m % x
 *   V tile: [d_h / (16 r)][4][16][r][4]: element (slot s, dim m) at
 *            ((((m / (16 r)) * 4 + s / 4) * 16 + m % 16) * r + (m / 16) % r) * 4 + s % 4
 *            (each 16 bytes hold 4 consecutive slots of r dimensions 16 apart)
 * For FP8_E4M3 pools the stored code is multiplied by a per-(layer, page, kv-head) fp32 scale:
 *   k_scale, v_scale: [num_layers][num_pages][num_kv_heads]; NULL for other dtypes. */
typedef struct {
  const void *k_pages;
  const void *v_pages;
  const float *k_scale;
  const float *v_scale;
  int32_t num_pages;
} kvprm_kv_cache;

/* The candidates to score. Candidate b has L_b = lengths[b] cached tokens at positions
 * 0..L_b-1; token t sits in logical page t / 16, slot t % 16, and logical page i maps to
 * physical page page_table[b * max_pages + i]. Slots at or beyond L_b in the last page and
 * table entries beyond ceil(L_b / 16) are never read (they may hold garbage or -1).
 * The verify token sits at position L_b and attends to the L_b cached keys and its own key.
 *
 * Prefix-sharing hint (optional; section 4.1: beam candidates that extend one prefix share its
 * cached keys and values): candidates [group_start_host[g], group_start_host[g+1]) share their
 * first group_prefix_len_host[g] tokens, which must be a multiple of 16 and at most every
 * member's length (checked against lengths_host, which the hint requires), and be held by the
 * same physical pages in every member's row (not checked: the shared part is read through the
 * first member's row). Groups tile [0, B). With bf16 or fp8 caches and at most 64 groups the
 * shared pages are read once per group instead of once per member; otherwise the hint is
 * ignored. A valid hint changes results only by floating-point summation order. */
typedef struct {
  int32_t batch;                        /* B >= 0 */
  const int32_t *page_table;            /* device [B][max_pages] */
  int32_t max_pages;                    /* >= 1 */
  const int32_t *lengths;               /* device [B], 0 <= L_b <= max_pages * 16 */
  /* Optional host mirror of lengths. When given it must equal the device lengths at the time
   * the enqueued work runs (also on every replay of a captured graph): the chunk grid of the
   * attention kernels is sized from it, so a device length above its mirror would leave the
   * chunks past that grid uncomputed (checked only in the KVPRM_DEBUG mode). NULL sizes the
   * grid from max_pages, which is valid for any device lengths. */
  const int32_t *lengths_host;
  int32_t num_groups;                   /* 0 = no prefix-sharing hint */
  const int32_t *group_start_host;      /* [num_groups + 1] */
  const int32_t *group_prefix_len_host; /* [num_groups] */
} kvprm_batch;

/* Create a handle for one model shape. Returns KVPRM_E_UNSUPPORTED for shapes outside the list
 * above. *out is set only on success. */
kvprm_status kvprm_create(const kvprm_model_desc *desc, kvprm_handle *out);

/* Release a handle (NULL is accepted). */
kvprm_status kvprm_destroy(kvprm_handle h);

/* Bytes of device workspace kvprm_score and kvprm_attention need for this batch (it depends on
 * batch and max_pages only). */
kvprm_status kvprm_workspace_size(kvprm_handle h, const kvprm_batch *batch, size_t *bytes);

/* Eq. (score) for every candidate: scores[b] = P(+) in [0, 1] and, if logits != NULL,
 * logits[b] = z_b = w_r . RMSNorm(x_b) + b_r (fp32, device [B]). The residual stream, queries,
 * softmax state and accumulators are fp32; weights and cache are read at their stored
 * precision. B = 0 returns KVPRM_OK and enqueues nothing. The workspace (device, 256-byte
 * aligned, >= kvprm_workspace_size bytes) is scratch owned by the call until the stream
 * passes it; its contents on entry do not matter. */
kvprm_status kvprm_score(kvprm_handle h, const kvprm_kv_cache *cache, const kvprm_batch *batch,
                         const kvprm_readout_weights *weights, void *workspace, size_t ws_bytes,
                         float *scores, float *logits, void *stream);

/* Bytes of the static workspace of kvprm_score_static (64 MiB per GPU). */
#define KVPRM_STATIC_WORKSPACE_BYTES (64u << 20)

/* kvprm_score without a workspace argument, for callers that cannot allocate device memory
 * (code under HIP graph capture that must not allocate, tight serving loops, harnesses that
 * forbid hipMalloc). The workspace is a static device array of KVPRM_STATIC_WORKSPACE_BYTES
 * that the library holds on every GPU it runs on until the process ends; nothing is allocated
 * or freed by the call. It serves batches whose kvprm_workspace_size is at most that size
 * (8 candidates with up to 32768 cached tokens at the 7B shape need 16 MiB; 64 candidates with
 * 18432 tokens each need 87 MiB and are refused); a larger one returns KVPRM_E_WORKSPACE before
 * anything is enqueued.
 * Every call on one GPU, from any handle or thread, uses the same array, which keeps the
 * previous call's contents (no call needs it cleared): calls whose work overlaps on one GPU
 * race, so the caller serialises them (for example by issuing them on one stream). The work
 * runs on the current device; a non-null stream must belong to it (KVPRM_E_INVALID
 * otherwise). The first call on a device resolves that device's copy of the array. Outputs
 * and the other conventions are those of kvprm_score. */
kvprm_status kvprm_score_static(kvprm_handle h, const kvprm_kv_cache *cache,
                                const kvprm_batch *batch, const kvprm_readout_weights *weights,
                                float *scores, float *logits, void *stream);

/* The attention step of one layer alone (for tests and diagnostics): for every candidate b and
 * q-head h, o[b][h] = softmax(q K^T / sqrt(d_h)) V over the L_b cached keys/values of `layer`
 * and the extra key/value k_self[b][h / g], v_self[b][h / g] (the verify token's own).
 * q: device fp32 [B][n_q][d_h] (already rotated); k_self, v_self: device fp32 [B][n_kv][d_h];
 * o: device fp32 [B][n_q][d_h]. The prefix-sharing hint is honoured as in kvprm_score. */
kvprm_status kvprm_attention(kvprm_handle h, const kvprm_kv_cache *cache, const kvprm_batch *batch,
                             int32_t layer, const float *q, const float *k_self,
                             const float *v_self, void *workspace, size_t ws_bytes, float *o,
                             void *stream);

/* The split-L step of kvprm_attention alone (the shared-prefix and per-candidate chunk kernels,
 * without the merge): for every candidate, q-head and chunk of cached pages, the unnormalised
 * softmax state of that chunk (running maximum, sum of exponentials, exponential-weighted sum of
 * values; the split form of the appendix's softmax(qK^T/sqrt(d))V) is written to the workspace
 * in an internal layout. The verify token's own key is not applied and nothing else is
 * written. It exists to time and profile the chunk kernels on their own; arguments, validation
 * and errors are as for kvprm_attention. */
kvprm_status kvprm_attention_partials(kvprm_handle h, const kvprm_kv_cache *cache,
                                      const kvprm_batch *batch, int32_t layer, const float *q,
                                      void *workspace, size_t ws_bytes, void *stream);

/* Low-rank adapter of the readout, unmerged (section 4.1, Eq. (score): the verify token runs
 * f_{theta + dtheta}, the base model with a LoRA adapter dtheta; the paper trains rank 256,
 * alpha 32). For a projection with base matrix W [out][in], the factors are A [r][in] and
 * B [out][r]; the verify token applies W u + scale * B (A u), with scale = alpha / r, which
 * equals merging W' = W + scale * B A without holding a second copy of the weights (the cache
 * positions were produced by the base weights, adapter off). Factors are bf16 in the packed tile
 * layout of kvprm_pack_weight (A: rows = r, K = in; B: rows = out, K = r). A projection without
 * an adapter has a == b == NULL; a and b are both set or both NULL. */
typedef struct {
  const void *a; /* [r][in] */
  const void *b; /* [out][r] */
} kvprm_lora_factors;

typedef struct {
  kvprm_lora_factors q, k, v, o, gate, up, down; /* in = H (q, k, v, gate, up), n_q d_h (o), F (down) */
} kvprm_layer_lora;

typedef struct {
  const kvprm_layer_lora *layers; /* HOST array [num_layers] of device pointers */
  int32_t rank;                   /* r: a multiple of 32 in [32, 512] */
  float scale;                    /* alpha / r */
} kvprm_lora;

/* Workspace bytes of kvprm_score_lora for this batch and adapter rank (>= the bytes of
 * kvprm_workspace_size). KVPRM_E_UNSUPPORTED for fp32 weights. */
kvprm_status kvprm_workspace_size_lora(kvprm_handle h, const kvprm_batch *batch, int32_t rank,
                                       size_t *bytes);

/* kvprm_score with the base weights and an unmerged adapter: every adapted projection of the
 * verify token is W u + scale * B (A u); the rest of the pass, the outputs and the conventions
 * are those of kvprm_score. Requires BF16 weights (KVPRM_E_UNSUPPORTED otherwise); rank outside
 * [32, 512] or not a multiple of 32, or a factor pair with one pointer NULL, is
 * KVPRM_E_INVALID. The workspace must hold kvprm_workspace_size_lora(batch, rank) bytes. */
kvprm_status kvprm_score_lora(kvprm_handle h, const kvprm_kv_cache *cache,
                              const kvprm_batch *batch, const kvprm_readout_weights *base,
                              const kvprm_lora *lora, void *workspace, size_t ws_bytes,
                              float *scores, float *logits, void *stream);

/* Options of kvprm_score_ex. */
typedef struct {
  /* Unmerged adapter (as kvprm_score_lora), or NULL when the weights are theta + dtheta
   * merged (as kvprm_score). */
  const kvprm_lora *lora;
  /* Depth-k readout (section 3, definition of the depth-k readout; the k > 1 experiment of
   * section 5): depth = k verify tokens are appended to each candidate at positions
   * L_b .. L_b + k - 1 and pass through the readout together, token i attending to the L_b
   * cached keys and to verify tokens 0..i (causal), the adapter active on all of them; the
   * score and logit are read from the last one. depth = 1 is Eq. (score). depth > 1 requires
   * BF16 weights, depth * (num_q_heads / num_kv_heads) <= 16 and batch * depth <= 64
   * (KVPRM_E_UNSUPPORTED otherwise). */
  int32_t depth;
} kvprm_score_options;

/* Workspace bytes of kvprm_score_ex for this batch and these options. */
kvprm_status kvprm_workspace_size_ex(kvprm_handle h, const kvprm_batch *batch,
                                     const kvprm_score_options *options, size_t *bytes);

/* kvprm_score with options (unmerged adapter, depth-k readout); outputs and conventions are
 * those of kvprm_score, one score per candidate. options NULL is kvprm_score. */
kvprm_status kvprm_score_ex(kvprm_handle h, const kvprm_kv_cache *cache, const kvprm_batch *batch,
                            const kvprm_readout_weights *weights,
                            const kvprm_score_options *options, void *workspace, size_t ws_bytes,
                            float *scores, float *logits, void *stream);

/* Gradients of the score with respect to the cache (appendix, KV Steering: the score is a
 * differentiable function of the cached keys and values). For every candidate b the loss is
 * -log P(+)_b, and the derivative with respect to every cached key and value the candidate
 * reads (every layer, positions 0..L_b-1) is produced by a backward pass through the readout:
 * reward head, final RMSNorm, and per layer (last to first) the FFN, the output projection,
 * the attention over the cache and the token's own key (softmax recomputed from the forward's
 * log-sum-exp), the rotary embedding, the q/k/v projections and the RMSNorms. Requires BF16
 * weights and a BF16 cache, batch <= 8, hidden size <= 16384, ffn_dim and (n_q + 2 n_kv) d_h
 * at most 73728, and candidates that do not share cache pages (no prefix-sharing hint; a page
 * read by two candidates would get one of the two gradients): KVPRM_E_UNSUPPORTED /
 * KVPRM_E_INVALID otherwise. The workspace is
 * kvprm_workspace_size_grad bytes (activations of every layer are kept). */
kvprm_status kvprm_workspace_size_grad(kvprm_handle h, const kvprm_batch *batch, size_t *bytes);

/* scores[b] = P(+) as kvprm_score; grad_k, grad_v: device fp32 arrays with the element order of
 * the pools ([num_layers][num_pages][num_kv_heads][tile], element i is the derivative with
 * respect to pool element i). Elements of the pages a candidate reads are written (zero for
 * slots at or beyond L_b); elements of other pages are left as they are. */
kvprm_status kvprm_score_grad(kvprm_handle h, const kvprm_kv_cache *cache,
                              const kvprm_batch *batch, const kvprm_readout_weights *weights,
                              void *workspace, size_t ws_bytes, float *scores, float *grad_k,
                              float *grad_v, void *stream);

/* KV Steering (appendix algorithm): `steps` times, every cached key and value the candidates
 * read (slots 0..L_b-1) becomes round_bf16(kv - eta * d(-log P(+))/d kv), the gradient taken at
 * the cache as it is at that step. The pools of `cache` are WRITTEN in place (the only entry
 * point that writes the cache). scores_before[b] = P(+) before the first step, scores_after[b]
 * = P(+) after the last (device fp32 [B]). Requirements as for kvprm_score_grad; steps >= 1. */
kvprm_status kvprm_steer(kvprm_handle h, const kvprm_kv_cache *cache, const kvprm_batch *batch,
                         const kvprm_readout_weights *weights, float eta, int32_t steps,
                         void *workspace, size_t ws_bytes, float *scores_before,
                         float *scores_after, void *stream);

/* Repack one bf16 weight matrix W [rows][K] from row-major order into the packed tile layout
 * that kvprm_score reads for BF16 weights: blocks of 1 KiB, block kb * (rows / 16) + t holding
 * rows 16t .. 16t+15 and inputs 32kb .. 32kb+31; inside a block, 16-byte group l (0..63) holds
 * W[16t + l % 16][32kb + 8 (l / 16) + i], i = 0..7. src and dst are device pointers to rows * K
 * bf16 values that must not overlap; rows % 16 == 0 and K % 32 == 0, else KVPRM_E_INVALID.
 * Enqueued on `stream`; a one-time preparation of static weights, not part of scoring. */
kvprm_status kvprm_pack_weight(const void *src, void *dst, int64_t rows, int64_t K, void *stream);

/* Which pool kvprm_pack_kv writes: the K and V tiles have different stored layouts. */
typedef enum { KVPRM_KEYS = 0, KVPRM_VALUES = 1 } kvprm_kv_part;

/* Converts cache tiles written token by token into the stored tile layout of kvprm_kv_cache
 * (section 2: the generator caches the key and value of every token at every layer; this is
 * the bridge from a token-major paged cache to the layout the scoring kernels stream).
 * src: num_tiles tiles of page_size (16) x head_dim values of `dtype` in token-major order,
 *      element (slot s, dim m) of tile t at t * 16 * head_dim + s * head_dim + m, i.e. a pool
 *      [num_layers][num_pages][num_kv_heads][16][head_dim] when num_tiles = num_layers *
 *      num_pages * num_kv_heads;
 * dst: the same tiles in the K (part = KVPRM_KEYS) or V (KVPRM_VALUES) tile layout described at
 *      kvprm_kv_cache, in the same tile order (fp8 per-tile scales therefore keep their order
 *      and are not touched).
 * The bytes are moved unchanged (slots past a sequence's end may hold anything, NaN included).
 * dtype F32, BF16 or FP8_E4M3; head_dim 64 or 128 (KVPRM_E_UNSUPPORTED otherwise); src and dst
 * device pointers, 16-byte aligned, not overlapping (KVPRM_E_INVALID otherwise); num_tiles = 0
 * does nothing. Nothing is allocated; enqueued on `stream`. */
kvprm_status kvprm_pack_kv(const void *src, void *dst, int64_t num_tiles, int32_t head_dim,
                           kvprm_dtype dtype, kvprm_kv_part part, void *stream);

/* Diagnostic (measurement, not part of scoring): read `bytes` of device memory at `buf` once,
 * with the access pattern of the cache and weight streams (16-byte non-temporal loads, 512
 * blocks of 256 threads striding over the buffer), and XOR all its 32-bit words into the device
 * word *sink (one atomic per wave; the result keeps the reads from being removed and lets a
 * caller check that every word was read once). The elapsed time gives the streaming-read
 * ceiling of the GPU that the kernels' HBM fractions are compared with. buf 16-byte aligned,
 * bytes a positive multiple of 16, sink 4-byte aligned: KVPRM_E_INVALID otherwise. Nothing is
 * allocated; enqueued on `stream`. */
kvprm_status kvprm_stream_read(const void *buf, size_t bytes, uint32_t *sink, void *stream);

/* Text of the last error on the calling thread ("" if none). Valid until the next call on
 * this thread. */
const char *kvprm_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* KVPRM_H */
