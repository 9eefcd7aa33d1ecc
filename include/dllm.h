/*
 * dllm.h - C ABI of the MI355X (gfx950) denoising-step library (libdllm.so).
 *
 * Block-wise diffusion-LLM inference (paper: Background, "Block-Wise Decoding"):
 * the output is split into consecutive blocks decoded left to right.  At each
 * denoising step the transformer runs over the current decoding window (the
 * current block, optionally extended with speculative draft tokens of the next
 * block; System Design, "Multi-Block Speculative Decoding"), attending to a
 * reused prefix KV cache and globally within the window, and every masked
 * position gets a predicted id and a confidence; a confidence-selected subset is
 * committed.  Completed blocks are appended to the prefix cache; revised prefix
 * positions can have their KV refreshed sparsely (System Design, "Dual-Path
 * Progressive Revision", "Sparse Cache Refresh"), visible from the next step on.
 *
 * Model: pre-norm LLaMA-style blocks (RMSNorm, multi-head attention with
 * rotate-half RoPE, SwiGLU FFN, no biases) and an untied LM head, as the paper's
 * operator list (RMSNorm, matrix multiplication, FlashAttention, elementwise ops;
 * Implementation section) and the LLaDA-8B model it evaluates imply.  For the
 * Dream-7B model of its cross-model study (Evaluation: grouped-query attention with
 * fewer K/V heads) a config may give fewer K/V heads than query heads (query head h
 * reads K/V head h / (n_heads / n_kv_heads)) and biases on the Q/K/V projections.
 *
 * Conventions
 *  - Every function returns an int status: DLLM_OK (0) or a negative DLLM_E_*.
 *    dllm_last_error() returns a thread-local message for the last failure.
 *    No C++ exception crosses this boundary.
 *  - Arguments are validated on the host before any GPU work is queued; a call
 *    that fails validation queues nothing and changes no state.
 *  - Device work is asynchronous on the given stream (a hipStream_t; NULL is
 *    the null stream).  Outputs are valid once that stream has completed.
 *    The host-side prefix length of a KV handle changes when the call returns.
 *  - "d_" pointers are device pointers; the caller owns them and they must stay
 *    valid until the stream work that uses them has finished.  The library owns
 *    only its handles, its prepacked weight copy and its workspaces, all freed by
 *    the matching *_destroy call.
 *  - A model handle is not thread-safe: calls that use one model must not run
 *    concurrently (they share the model's workspaces), and all its calls should
 *    be issued on one stream, or on streams the caller orders.
 *
 * Readings where the paper is silent (also fixed by the test oracle):
 *  - confidence = softmax probability of the argmax token (temperature 0); the
 *    MASK id is excluded from argmax and softmax; argmax ties -> lowest id;
 *  - commit order: higher confidence first, equal confidence -> lower position;
 *  - the prefix is block-causal: the prompt is one bidirectional block, block b
 *    sees blocks <= b; a denoising window sees every key in [0, P + W).
 */
#ifndef DLLM_H
#define DLLM_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define DLLM_OK 0
#define DLLM_E_INVAL (-1)     /* bad argument (null pointer, out-of-range size, ...) */
#define DLLM_E_CAPACITY (-2)  /* the KV cache or a window limit would overflow */
#define DLLM_E_DTYPE (-3)     /* unsupported dtype / shape combination */
#define DLLM_E_HIP (-4)       /* a HIP runtime call failed */
#define DLLM_E_UNIMPL (-5)    /* not implemented for this configuration */
#define DLLM_E_NOMEM (-6)     /* device allocation failed */

/* Weight / arithmetic types. */
#define DLLM_F32 0   /* fp32 weights, fp32 activations and KV cache */
#define DLLM_BF16 1  /* bf16 weights; GEMM activations as bf16 hi/lo pairs, Q as fp16 hi/lo, KV cache fp16; fp32 accumulate */
#define DLLM_W8 2    /* int8 weights with fp32 per-output-row scales; activations as for DLLM_BF16 */
#define DLLM_Q4 3    /* Q4_0 weights (see dllm_quantize_q4_0); activations as for DLLM_BF16 */

typedef struct dllm_model dllm_model;
typedef struct dllm_kv dllm_kv;
typedef void* dllm_stream; /* hipStream_t */

typedef struct dllm_config {
    int32_t n_layers;
    int32_t d_model;     /* = n_heads * head_dim */
    int32_t n_heads;
    int32_t head_dim;    /* 64 or 128 */
    int32_t d_ff;        /* SwiGLU hidden size */
    int32_t vocab;
    int32_t mask_id;     /* id of the MASK token, 0 <= mask_id < vocab */
    int32_t block;       /* block size of the block-causal prefix (32) */
    float eps;           /* RMSNorm epsilon */
    float rope_base;     /* RoPE base (10000) */
    int32_t dtype;       /* DLLM_F32, DLLM_BF16, DLLM_W8 or DLLM_Q4 */
    int32_t max_window;  /* largest row count of a step / append / refresh call (<= 256) */
    int32_t max_pos;     /* positions covered by the RoPE table; bounds every KV capacity */
    int32_t n_kv_heads;  /* K/V heads (grouped-query attention); 0 = n_heads; must divide n_heads */
    int32_t qkv_bias;    /* 1: the Q/K/V projections have fp32 biases (bq, bk, bv); else 0 */
} dllm_config;

/* Device pointers to row-major [out][in] matrices of one layer.
 * DLLM_F32: float; DLLM_BF16, DLLM_W8 and DLLM_Q4: bfloat16 (W8 and Q4 quantise them
 * on create).
 * wq, wo: [d][d]; wk, wv: [dkv][d] with dkv = n_kv_heads * head_dim; wg, wu:
 * [d_ff][d]; wd: [d][d_ff]; norms: float [d]; biases (read only when
 * cfg.qkv_bias, else may be NULL): float bq [d], bk [dkv], bv [dkv]. */
typedef struct dllm_layer_weights {
    const void* wq;
    const void* wk;
    const void* wv;
    const void* wo;
    const void* wg;
    const void* wu;
    const void* wd;
    const float* attn_norm;
    const float* ffn_norm;
    const float* bq;
    const float* bk;
    const float* bv;
} dllm_layer_weights;

typedef struct dllm_weights {
    const void* embed;                 /* [vocab][d]: float (F32) or bfloat16 (BF16, W8) */
    const void* lm_head;               /* [vocab][d], same type as the layer matrices */
    const float* final_norm;           /* [d] */
    const dllm_layer_weights* layers;  /* HOST array of n_layers entries */
} dllm_weights;

/* Message of the last failed call on this thread ("" if none). */
const char* dllm_last_error(void);

/* Library version string. */
const char* dllm_version(void);

/* Creates a model: validates the config, allocates the library's own copy of the
 * weights prepacked into MFMA-fragment order (and, for DLLM_W8, quantises every
 * matrix except the embedding to int8 with per-output-row fp32 scales
 * s = max|w| / 127, q = round-half-even(w / s), decided in fp32; for DLLM_Q4, to
 * Q4_0 as dllm_quantize_q4_0 does, and the matrix products then use the weights
 * (q - 8) * d exactly, with no rounding of the dequantised values), builds the
 * RoPE table, and allocates workspaces for max_window rows.  The caller's weight
 * buffers are only read during this call (on `stream`, which is synchronised
 * before returning) and may be freed afterwards.  Quantisation is the analog of
 * the paper's converter layout pass (Implementation section). */
int dllm_model_create(const dllm_config* cfg, const dllm_weights* w, dllm_stream stream,
                      dllm_model** out);
int dllm_model_destroy(dllm_model* m);

/* Bytes of device memory a KV cache of `capacity` positions needs (4 bytes per
 * cached value for DLLM_F32 models, 2 otherwise).  Layout inside the caller's
 * buffer, with Cs = capacity rounded up to a multiple of 32, H = n_kv_heads (n_heads
 * if 0) and P = H*Cs*Dh elements per plane, 2 planes per layer (K, V^T):
 *     K   of layer l, head h, position p, dim j: (l*2+0)*P + (h*Cs + p)*Dh + j
 *     V^T of layer l, head h, dim j, position p: (l*2+1)*P + (h*Dh + j)*Cs + p
 * Elements are float for DLLM_F32 models and IEEE fp16 (round to nearest even,
 * saturated at +-65504) for DLLM_BF16, DLLM_W8 and DLLM_Q4 models.  K is stored after
 * RoPE. */
int dllm_kv_bytes(const dllm_model* m, int32_t capacity, size_t* bytes);

/* Wraps a caller-owned device buffer of at least dllm_kv_bytes() bytes as a KV
 * cache (borrowed, not freed by the library).  prefix_len starts at 0.
 * capacity must be <= cfg.max_pos. */
int dllm_kv_create(const dllm_model* m, void* d_buf, size_t bytes, int32_t capacity, dllm_kv** out);
int dllm_kv_destroy(dllm_kv* kv);
int dllm_kv_prefix_len(const dllm_kv* kv, int32_t* prefix_len, int32_t* prompt_len);
/* Rewinds (or restores) the prefix length, e.g. to repeat an identical step.
 * Requires prompt_len <= prefix_len <= capacity; rows past it are ignored. */
int dllm_kv_set_prefix_len(dllm_kv* kv, int32_t prefix_len);

/* Prompt processing (Evaluation setup: latency includes prompt processing).
 * Runs the n prompt ids through every layer as one bidirectional block at
 * positions [0, n) and writes their K/V.  Requires prefix_len == 0; sets
 * prefix_len = prompt_len = n.  E_CAPACITY if n > capacity.  Ids outside
 * [0, vocab) are read as the MASK id. */
int dllm_prefill(dllm_model* m, dllm_kv* kv, const int32_t* d_ids, int32_t n, dllm_stream stream);

/* One denoising step over the W-row window at positions [P, P + W), P = prefix_len
 * (Background, "Block-Wise Decoding"; System Design, "Multi-Block Speculative
 * Decoding").  Row i feeds the MASK id if d_mask[i] != 0, else d_tok[i]; every
 * row attends to all keys [0, P + W) (the whole prefix and the window, both
 * directions).  Writes, for every row, the argmax id (MASK excluded, lowest id on
 * ties) to d_out_id[W] and its softmax probability to d_out_conf[W].  Logits never
 * reach device memory.  The window's K/V are written to cache rows [P, P + W),
 * which stay scratch (prefix_len is unchanged), so draft rows never enter the
 * prefix.  E_INVAL if W < 1 or W > max_window; E_CAPACITY if P + W > capacity. */
int dllm_denoise_step(dllm_model* m, dllm_kv* kv, const int32_t* d_tok, const uint8_t* d_mask,
                      int32_t W, int32_t* d_out_id, float* d_out_conf, dllm_stream stream);

/* dllm_denoise_step for callers that cannot allocate device memory: code under HIP
 * graph capture, tight serving loops, harnesses that forbid hipMalloc.  Same
 * arguments, checks and results as dllm_denoise_step, but the step's scratch (the
 * residual stream, activation fragments, split-K, attention and LM-head partials)
 * is carved from a static device array of the library (64 MiB per device, held until
 * the process ends) instead of the model's workspace; the call itself allocates and
 * frees nothing.  The array's device address is resolved once per device (at
 * dllm_model_create, or at the first call on a device).  Every call on a device
 * shares that device's array and leaves the last call's contents in it: calls that
 * overlap on one device (concurrent streams, threads, or this call beside another
 * model's) race.  Each call first clears what must be zero (the padding columns of
 * its activation fragments, when d_model or d_ff is not a whole number of 32- or
 * 64-column chunks; no launch otherwise); every other buffer the step reads is
 * written by the same step first, or feeds only padding rows.  E_CAPACITY if the
 * step's scratch for this model and W exceeds 64 MiB (LLaDA-8B and Dream-7B widths
 * need about 40 MiB at W <= 64), plus dllm_denoise_step's errors. */
int dllm_denoise_step_noalloc(dllm_model* m, dllm_kv* kv, const int32_t* d_tok, const uint8_t* d_mask, int32_t W,
                              int32_t* d_out_id, float* d_out_conf, dllm_stream stream);

/* Confidence-selected commit over one segment (Background: "updates a
 * confidence-selected subset"; a draft segment is committed separately, System
 * Design, "Multi-Block Speculative Decoding").  Among the positions p in
 * [seg_begin, seg_begin + seg_len) with d_mask[p] != 0, takes the k with the
 * highest d_conf (ties -> lower position), sets d_tok[p] = d_id[p] and
 * d_mask[p] = 0.  Writes the committed positions, in that order, to
 * d_committed_pos[0 .. n) and n = min(k, #masked) to *d_n_committed.
 * d_committed_pos must hold min(k, seg_len) entries; it and d_n_committed may be
 * NULL.  E_INVAL if k < 0, seg_begin < 0, seg_len < 0 or seg_len > 1024. */
int dllm_commit(const float* d_conf, const int32_t* d_id, int32_t* d_tok, uint8_t* d_mask,
                int32_t seg_begin, int32_t seg_len, int32_t k, int32_t* d_committed_pos,
                int32_t* d_n_committed, dllm_stream stream);

/* Appends a completed block (Background, "Block-Wise Decoding": completed blocks
 * are reused through the KV cache).  Its n ids run through every layer at
 * positions [P, P + n), attending to keys [0, P + n); their K/V are written and
 * prefix_len becomes P + n.  The ids must hold no MASK.  E_INVAL if n < 1 or
 * n > max_window; E_CAPACITY if P + n > capacity. */
int dllm_append_prefix_kv(dllm_model* m, dllm_kv* kv, const int32_t* d_block_tok, int32_t n,
                          dllm_stream stream);

/* Sparse KV refresh of revised prefix positions (System Design, "Sparse Cache
 * Refresh": confidence, identity and KV of revisable tokens are recomputed and
 * merged at a step boundary).  Each of the n rows runs its new id d_new_id[i] at
 * position d_pos[i]; at every layer the new K/V of all n rows replace the cached
 * ones before that layer's attention, and row i attends to keys [0, e_i), e_i the
 * end of its block (prompt: prompt_len; else prompt_len + block * (1 + (p -
 * prompt_len) / block)), capped at prefix_len.  Every other cached row is left as
 * it was.  If d_out_id / d_out_conf are non-NULL, also writes the rows' argmax id
 * and confidence.  The positions are copied to the host (the call synchronises
 * `stream`) to validate them: E_INVAL unless all are distinct and < prefix_len,
 * n >= 1 and n <= max_window. */
int dllm_refresh_kv(dllm_model* m, dllm_kv* kv, const int32_t* d_pos, const int32_t* d_new_id,
                    int32_t n, int32_t* d_out_id, float* d_out_conf, dllm_stream stream);

/* Piggybacked append and refresh: one forward over three row groups that is, row
 * for row, the sequence dllm_refresh_kv(ref) -> dllm_append_prefix_kv(block) ->
 * dllm_denoise_step(window) (System Design, "Sparse Cache Refresh": revisions are
 * merged at step boundaries; "Multi-Block Speculative Decoding": a completed
 * block becomes prefix before the next step), streaming the weights once instead
 * of three times:
 *   - rows [0, n_ref): revised prefix positions d_ref_pos[i] with ids d_ref_id[i]
 *     (as dllm_refresh_kv: keys up to the end of their block, capped at P, the
 *     prefix length on entry; their new K/V replace the cached ones layer by
 *     layer);
 *   - rows [n_ref, n_ref + n_block): the completed block d_block_tok (no MASK) at
 *     positions P.., keys [0, P + n_block), written into the prefix;
 *   - the last W rows: the window d_tok / d_mask (nullable) at positions
 *     P + n_block.., keys [0, P + n_block + W), as dllm_denoise_step.
 * A refresh position inside the block being appended is expressed by appending
 * the block with the revised id.  The LM head runs only over the rows whose
 * outputs are asked for (never the appended block's).  Outputs (each pair both set
 * or both NULL):
 * d_out_id / d_out_conf [W] for the window, d_ref_out_id / d_ref_out_conf [n_ref]
 * for the refresh rows.  prefix_len becomes P + n_block.  Any group may be empty;
 * E_INVAL unless 1 <= n_ref + n_block + W <= max_window and the refresh positions
 * are distinct and < P (they are copied to the host, so the call synchronises
 * `stream` when n_ref > 0); E_CAPACITY if P + n_block + W > capacity. */
int dllm_step_merged(dllm_model* m, dllm_kv* kv, const int32_t* d_ref_pos, const int32_t* d_ref_id,
                     int32_t n_ref, const int32_t* d_block_tok, int32_t n_block, const int32_t* d_tok,
                     const uint8_t* d_mask, int32_t W, int32_t* d_out_id, float* d_out_conf,
                     int32_t* d_ref_out_id, float* d_ref_out_conf, dllm_stream stream);

/* A denoising step over a decoding window that has slid past committed positions
 * (System Design, "Multi-Block Speculative Decoding": the window, not the block,
 * is the execution unit and moves with the commit frontier).  The W rows sit at
 * positions [w0, w0 + W) with w0 >= prefix_len and attend to every key in
 * [0, w0 + W); rows [prefix_len, w0) are positions an earlier window step wrote
 * and are reused as they are (the caller keeps them current).  Their K/V land in
 * rows [w0, w0 + W).  Outputs as dllm_denoise_step; prefix_len is unchanged.
 * With w0 = prefix_len this is dllm_denoise_step.  E_INVAL if W is not in
 * [1, max_window] or w0 < prefix_len; E_CAPACITY if w0 + W > capacity. */
int dllm_denoise_window(dllm_model* m, dllm_kv* kv, int32_t w0, const int32_t* d_tok,
                        const uint8_t* d_mask, int32_t W, int32_t* d_out_id, float* d_out_conf,
                        dllm_stream stream);

/* dllm_denoise_window with selective logits skipping (System Design, "Dual-Path
 * Progressive Revision", "Selective Logits Skipping": the output projection, the
 * confidence and the selection are computed only for positions whose identity or
 * confidence can still change a decision; stable positions skip them).  The
 * forward and the K/V it writes are dllm_denoise_window's.  d_need (device, W
 * bytes; NULL = every row) flags the rows that need an output, e.g. the mask of a
 * top-k step (committed rows are final) or the non-stable rows of a staged step.
 * The LM head then runs over at most n_need rows, the first flagged ones in row
 * order, packed together, so its cost follows n_need rather than W; each of those
 * rows gets the (id, conf) dllm_denoise_window would give it, every other row gets
 * id -1 and conf 0.  n_need = 0 skips the LM head.  E_INVAL unless
 * 0 <= n_need <= W, plus dllm_denoise_window's checks. */
int dllm_denoise_window_sls(dllm_model* m, dllm_kv* kv, int32_t w0, const int32_t* d_tok,
                            const uint8_t* d_mask, const uint8_t* d_need, int32_t n_need, int32_t W,
                            int32_t* d_out_id, float* d_out_conf, dllm_stream stream);

/* Parity only (never on the timed path): the same step as dllm_denoise_step, also
 * writing the full logits d_logits[W][vocab] (float, MASK column = -inf).  If
 * d_out_id / d_out_conf are non-NULL they receive the step's outputs. */
int dllm_debug_logits(dllm_model* m, dllm_kv* kv, const int32_t* d_tok, const uint8_t* d_mask,
                      int32_t W, float* d_logits, int32_t* d_out_id, float* d_out_conf,
                      dllm_stream stream);

/* Parity only: runs the window through the first n_layers layers (0 = embedding
 * only) and copies the fp32 residual stream to d_x[W][d_model]. */
int dllm_debug_hidden(dllm_model* m, dllm_kv* kv, const int32_t* d_tok, const uint8_t* d_mask,
                      int32_t W, int32_t n_layers, float* d_x, dllm_stream stream);

/* Kernel timing probe.  Kernel classes: */
#define DLLM_K_QKV 0
#define DLLM_K_ATTN 1
#define DLLM_K_OPROJ 2
#define DLLM_K_GATEUP 3
#define DLLM_K_DOWN 4
#define DLLM_K_LMHEAD 5
/* While enabled, every launch of `kernel_class` (at most max_records of them) is
 * bracketed by HIP events recorded on the launch stream.  kernel_class < 0
 * disables.  Recording the events adds small gaps, so timed throughput runs
 * should leave the probe disabled. */
int dllm_probe_enable(dllm_model* m, int32_t kernel_class, int32_t max_records);
/* Synchronises the recorded events and returns the count and mean duration
 * (milliseconds) of the recorded launches; resets the record count. */
int dllm_probe_read(dllm_model* m, int32_t* n_records, double* mean_ms);

/* Kernel timing by replay: issues, back to back on `stream`, n_launches launches of
 * one kernel class exactly as a denoising step over W rows at prefix P = prefix_len
 * issues them (same kernels, launch shapes and operands), layer 0, 1, ... cyclically
 * (the LM head: the same launch n_launches times).  The caller brackets the call
 * with events; elapsed / n_launches is the class's mean launch duration without
 * per-launch event records.  The operands are whatever the model's workspaces
 * hold (run a step first for realistic values); the launches overwrite those
 * workspaces and the cache rows [P, P + W) of every layer, which are step scratch,
 * and nothing else.  E_INVAL for an unknown class, W outside [1, max_window] or
 * n_launches < 1; E_CAPACITY if P + W > capacity. */
int dllm_kernel_replay(dllm_model* m, dllm_kv* kv, int32_t kernel_class, int32_t W, int32_t n_launches,
                       dllm_stream stream);

/* Algorithmic bytes one launch of a kernel class moves for a window of W rows at
 * prefix P: every weight once (with int8 row scales, Q4_0 block scales, Q/K/V
 * biases), the K/V the attention reads and the K/V rows QKV writes, one value per
 * element (4 bytes for DLLM_F32 models, 2 otherwise); no activations (L2-resident) and
 * no logits.  Used to express achieved bandwidth against the HBM roofline. */
int dllm_kernel_bytes(const dllm_model* m, int32_t kernel_class, int32_t W, int32_t P, double* bytes);

/* Token states of staged stabilisation (one byte per window position). */
#define DLLM_TOKEN_INVISIBLE 0  /* masked, or predicted with too little confidence: not context */
#define DLLM_TOKEN_VISIBLE 1    /* exposed to later steps as context, still revisable */
#define DLLM_TOKEN_STABLE 2     /* reliable enough for long-term reuse */

/* Staged token stabilisation for one segment [seg_begin, seg_begin + seg_len) of
 * the window (System Design, "Staged Token Stabilization"; the Evaluation setup
 * uses theta_visible 0.7 and theta_stable 0.9), a variant of dllm_commit:
 *   - every INVISIBLE position with conf >= theta_visible becomes VISIBLE: d_tok
 *     takes its predicted id and its mask flag is cleared;
 *   - if none does and INVISIBLE positions remain, the most confident of them
 *     becomes VISIBLE (equal conf: the lower position), so decoding progresses;
 *   - every VISIBLE position (just promoted or earlier) with conf >= theta_stable
 *     becomes STABLE.  A VISIBLE position keeps its id: identity revision goes
 *     through dllm_refresh_kv.
 * d_state (device, one byte per window position) holds the states and is
 * updated in place; positions outside the segment are untouched.  Comparisons
 * are in fp32.  d_promoted_pos (nullable, >= seg_len entries) receives the
 * positions that left INVISIBLE in ascending order, d_n_promoted (nullable) their
 * count.  Requires 1 <= seg_len <= 1024, seg_begin >= 0 and finite thresholds;
 * E_INVAL otherwise, before any launch.  Asynchronous on `stream`. */
int dllm_commit_staged(const float* d_conf, const int32_t* d_id, int32_t* d_tok, uint8_t* d_mask,
                       uint8_t* d_state, int32_t seg_begin, int32_t seg_len, float theta_visible,
                       float theta_stable, int32_t* d_promoted_pos, int32_t* d_n_promoted, dllm_stream stream);

/* Draft acceptance (System Design, "Multi-Block Speculative Decoding": when a
 * future block becomes current its draft tokens are re-evaluated and accepted only
 * if they meet the commitment criterion).  Over n position-aligned entries: every
 * position with d_mask = 1, d_draft_id >= 0, d_id == d_draft_id and
 * d_conf >= theta (fp32) is committed (d_tok = d_id, d_mask = 0).
 * d_accepted_pos (nullable, >= n entries) receives the accepted indices in
 * ascending order, d_n_accepted (nullable) their count.  E_INVAL unless
 * 1 <= n <= 1024 and theta is finite, before any launch. */
int dllm_accept_drafts(const float* d_conf, const int32_t* d_id, const int32_t* d_draft_id,
                       int32_t* d_tok, uint8_t* d_mask, int32_t n, float theta,
                       int32_t* d_accepted_pos, int32_t* d_n_accepted, dllm_stream stream);

/* Draft records for window rows past the current block: d_draft_id[i] = d_id[i]
 * where d_mask[i] = 1, else -1, for n position-aligned entries (n >= 1). */
int dllm_record_drafts(const int32_t* d_id, const uint8_t* d_mask, int32_t* d_draft_id, int32_t n,
                       dllm_stream stream);

/* Q4_0 quantisation, the converter step for DLLM_Q4 models (Implementation: the
 * operator library has a Q4_0 matrix multiplication and the model converter packs
 * quantised weights; Evaluation: every model runs Q4_0).  The GGUF Q4_0 format:
 * each row of the row-major [rows][K] source (float for src_dtype DLLM_F32,
 * bfloat16 for DLLM_BF16; device) is cut into nb = ceil(K / 32) blocks of 32
 * columns, a ragged last block padded with zeros.  Per block, in fp32: m = the
 * value of largest magnitude (the first in column order on ties) with its sign,
 * d = m / -8, inv = 1 / d (0 if d = 0), and every value x gets the code
 * q = min(15, trunc(x * inv + 8.5)); the weight it stands for is (q - 8) * d16
 * with d16 = d rounded to fp16 (nearest even).  Writes d_codes [rows][nb * 32]
 * (one code per byte, padding columns included) and d_scales [rows][nb] (fp16
 * bit patterns), both caller-owned device buffers, asynchronously on `stream`.
 * E_INVAL for NULL pointers or rows, K < 1; E_DTYPE for another src_dtype. */
int dllm_quantize_q4_0(const void* d_src, int32_t src_dtype, int32_t rows, int32_t K, uint8_t* d_codes,
                       uint16_t* d_scales, dllm_stream stream);

/* int8 quantisation, the converter step for DLLM_W8 models (Implementation: the
 * model converter packs quantised weights; the per-output-row int8 form is the
 * analog of the paper's Q4_0): for every row of the row-major [rows][K] source
 * (float for src_dtype DLLM_F32, bfloat16 for DLLM_BF16; device), in fp32:
 * s = max|w| / 127 and q = round-half-even(w / s) clamped to [-127, 127], both
 * divisions correctly rounded (a zero row gets s = 0 and codes 0); the weight q
 * stands for is q * s.  This is the quantiser dllm_model_create applies to DLLM_W8
 * models.  Writes d_codes [rows][K] and d_scales [rows] (caller-owned device
 * buffers) asynchronously on `stream`.  E_INVAL for NULL pointers or rows, K < 1;
 * E_DTYPE for another src_dtype. */
int dllm_quantize_int8(const void* d_src, int32_t src_dtype, int32_t rows, int32_t K, int8_t* d_codes,
                       float* d_scales, dllm_stream stream);

/* Measurement helper: one launch of a plain streaming read over `bytes` bytes of
 * the device buffer d_buf (16-byte aligned; bytes a multiple of 16), the same
 * 16-byte-per-lane non-temporal loads the GEMMs stream weights with.  The caller
 * times it with events on `stream` to measure the achievable HBM read rate that
 * the kernels' bandwidth is compared with.  d_sink (device, >= 4 bytes) receives a
 * value only in a case that never occurs for real data; it keeps the loads alive. */
int dllm_read_bandwidth(const void* d_buf, size_t bytes, uint32_t* d_sink, dllm_stream stream);

#ifdef __cplusplus
}
#endif

#endif /* DLLM_H */
