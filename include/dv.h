/*
 * dv.h - C ABI of the MI355X tree-verification library (libdv.so).
 *
 * One call runs the target model's parallel verification of a draft token
 * tree: the candidates go through the decoder stack in a single forward pass
 * over the committed KV cache, and the greedy acceptance rule picks the
 * accepted tokens, which then start the next round (Dovetail, arXiv
 * 2412.18934, Section 3.1 "CPU/GPU Heterogeneous Architecture"; greedy
 * exact-match verification per Section 5 "Verifying Draft Tokens").  The
 * verification latency T_V(gamma) this call realises is the quantity of
 * Section 2.2, eq. (speedup-breakdown), modelled in Appendix B as
 * max(T_c, T_p) + beta min(T_c, T_p).
 *
 * Conventions (the paper does not fix them; they are the standard Llama-2
 * decoder block read from the models of Section 4):
 *   - pre-norm RMSNorm, no biases, multi-head attention, SwiGLU FFN,
 *     rotary embedding with rotate-half pairing, untied lm_head, final norm;
 *   - every matrix is row-major [out][in]; activations are fp32;
 *   - tree node 0 is the root (the pending token), parents[0] = -1 and
 *     0 <= parents[i] < i for i >= 1; node i attends to every committed key
 *     plus its ancestors and itself and sits at position len + depth(i) - 1
 *     (root depth 1);
 *   - new keys/values are rounded to the cache dtype before any use;
 *   - argmax ties go to the lowest token id; the deepest accepted node wins,
 *     lowest node index on ties; the bonus token is the argmax at that node.
 *
 * Memory: the caller owns weights, KV buffers, logits and accept structs.
 * Device pointers are plain HIP device addresses (e.g. torch tensors'
 * data_ptr()).  The handle owns its workspace and frees it in
 * dv_verify_free; the library never frees caller memory.  A handle is bound
 * to one HIP stream and is not thread-safe.
 *
 * Errors: every call returns DV_OK (0) or a negative code.  Arguments are
 * validated before anything is launched, so a rejected call changes nothing
 * and the handle stays usable.  A HIP runtime failure returns DV_EHIP and
 * poisons the handle (every later call returns DV_EHIP).  dv_last_error
 * gives a message for the most recent failure.
 */
#ifndef DV_H
#define DV_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define DV_OK 0
#define DV_EINVAL (-1)    /* bad config, tree, token id, pointer or struct    */
#define DV_ECAPACITY (-2) /* len + n_tree exceeds the KV capacity or max_ctx  */
#define DV_ESTATE (-3)    /* commit without a matching pending step           */
#define DV_EHIP (-4)      /* HIP runtime error; sticky                        */
#define DV_ENOMEM (-5)    /* workspace allocation failed at init              */

#define DV_F32 0
#define DV_BF16 1
/* Weight-only int8 (the int8 setting the paper runs its target in on the
 * laptop, Section 4): every projection matrix (wq, wk, wv, wo, w_gate, w_up,
 * w_down, lm_head) is int8 [out][in] with one fp32 scale per output row,
 * W[r][c] = scale[r] * q[r][c]; the embedding, the norm gains and the KV
 * cache are bf16.  Activations and accumulation stay fp32 as for DV_BF16. */
#define DV_I8 2

#define DV_MAX_TREE 64

/* Model shape.  weight_dtype is also the KV-cache dtype (bf16 for DV_I8).
 * Shape limits: head_dim in {64, 128} with n_heads * head_dim == d_model;
 * d_model and vocab multiples of 32; d_ffn a multiple of 16;
 * 1 <= max_tree <= 64; for DV_I8, d_model and d_ffn multiples of 64. */
typedef struct dv_config {
    int32_t n_layers;
    int32_t d_model;
    int32_t n_heads;
    int32_t head_dim;
    int32_t d_ffn;
    int32_t vocab;
    float rms_eps;
    float rope_base;
    int32_t weight_dtype; /* DV_F32, DV_BF16 or DV_I8                        */
    int32_t max_ctx;      /* largest len + n_tree any step may reach          */
    int32_t max_tree;     /* largest n_tree (and prefill chunk), <= 64        */
} dv_config;

/* Device pointers to weights, all of weight_dtype (for DV_I8: projection
 * matrices int8, embed and norm gains bf16, plus the per-row scales).  The
 * per-layer fields are HOST arrays of n_layers device pointers; they are
 * copied at init, the weights themselves are not copied and must outlive the
 * handle.  The *_scale fields are read only for DV_I8 (NULL otherwise). */
typedef struct dv_weights {
    const void *embed;       /* [vocab][d_model]                 */
    const void *final_norm;  /* [d_model]                        */
    const void *lm_head;     /* [vocab][d_model]                 */
    const void *const *attn_norm; /* [d_model]                   */
    const void *const *wq;        /* [d_model][d_model]          */
    const void *const *wk;        /* [d_model][d_model]          */
    const void *const *wv;        /* [d_model][d_model]          */
    const void *const *wo;        /* [d_model][d_model]          */
    const void *const *ffn_norm;  /* [d_model]                   */
    const void *const *w_gate;    /* [d_ffn][d_model]            */
    const void *const *w_up;      /* [d_ffn][d_model]            */
    const void *const *w_down;    /* [d_model][d_ffn]            */
    const float *lm_head_scale;   /* [vocab]            (DV_I8)  */
    const float *const *wq_scale; /* [d_model] per layer (DV_I8) */
    const float *const *wk_scale; /* [d_model]                   */
    const float *const *wv_scale; /* [d_model]                   */
    const float *const *wo_scale; /* [d_model]                   */
    const float *const *w_gate_scale; /* [d_ffn]                 */
    const float *const *w_up_scale;   /* [d_ffn]                 */
    const float *const *w_down_scale; /* [d_model]               */
} dv_weights;

/* KV cache: device buffers of weight_dtype, per layer and head
 *   k: [n_layers][n_heads][capacity][head_dim]   (key-major rows)
 *   v: [n_layers][n_heads][capacity/32][head_dim][32]   (32-slot tiles:
 *      value (slot s, dim j) of a head at element ((s/32) head_dim + j) 32
 *      + s%32, so the 32 slots of a tile are one contiguous block, dim-major)
 * Slots [0, len) are committed.  capacity must be a positive multiple of 32
 * (DV_EINVAL otherwise).  len is host state that dv_kv_commit and
 * dv_prefill advance. */
typedef struct dv_kv {
    void *k;
    void *v;
    int32_t capacity;
    int32_t len;
} dv_kv;

/* Result of one verification step (host struct). */
typedef struct dv_accept {
    int32_t accept_len;             /* accepted nodes on the path, root included */
    int32_t path[DV_MAX_TREE];      /* node indices root -> deepest accepted     */
    int32_t bonus_token;            /* target's argmax at the last path node     */
    int32_t n_tree;                 /* step size, checked by dv_kv_commit        */
    int32_t base_len;               /* kv->len at the step, checked by commit    */
    int32_t argmax[DV_MAX_TREE];    /* per-node argmax of the logits             */
} dv_accept;

typedef struct dv_handle dv_handle;

/* Create a handle: validates cfg, copies the weight pointer tables, builds
 * the rotary cos/sin table (angles in double precision, stored fp32) and
 * allocates the workspace.  stream is a hipStream_t (NULL = default stream).
 * Returns DV_EINVAL, DV_ENOMEM or DV_EHIP on failure (*out set to NULL). */
int dv_verify_init(const dv_config *cfg, const dv_weights *w, void *stream, dv_handle **out);

/* One verification step over a draft tree (Section 3.1).
 *   tokens, tree_parents: HOST arrays of n_tree int32 (see tree contract);
 *   kv: the cache; the tree's keys/values are written to slots
 *       [len, len + n_tree); kv->len is not changed;
 *   out_logits: device [n_tree][vocab] fp32, or NULL to skip writing logits;
 *   out_accept: host struct, filled after the step completes (the call
 *       synchronises the handle's stream).
 * Repeating a step without committing recomputes the same result.
 * Errors: DV_EINVAL (tree, ids, pointers), DV_ECAPACITY, DV_EHIP. */
int dv_verify_step(dv_handle *h, const int32_t *tokens, const int32_t *tree_parents,
                   int32_t n_tree, dv_kv *kv, float *out_logits, dv_accept *out_accept);

/* Stochastic verification at temperature T > 0: the same forward pass as
 * dv_verify_step, then the speculative sampling rule instead of greedy
 * matching (Section 3.1 names speculative sampling as the acceptance rule;
 * Section 5 credits it with keeping the target's output distribution).  Reading: the
 * children of node u are independent draws from the draft distribution
 * draft_probs[u]; with p = softmax(logits[u] / T), starting at the root the
 * children of the current node are tried in index order; child c (token t)
 * is accepted when u_accept[c] * q[u][t] < p[t] and becomes the current
 * node; a rejected child replaces p by max(p - q[u], 0), renormalised; when
 * no child is accepted the bonus token is drawn from the current p by
 * inverse CDF (smallest id whose running mass exceeds u_bonus[current]
 * times the total).  All arithmetic is fp32.
 *   draft_probs: device [n_tree][vocab] fp32, 16-byte aligned, row u = the
 *       draft distribution at node u (rows of nodes without children are not
 *       read; entries must be >= 0, rows need not be normalised exactly);
 *   temperature: finite, > 0;
 *   u_accept, u_bonus: HOST arrays of n_tree floats in [0, 1) (the random
 *       numbers the rule draws; u_accept[0] is not used);
 *   out_logits: as dv_verify_step (16-byte aligned); when NULL the logits
 *       go to a workspace of the handle;
 *   other arguments as dv_verify_step.  out_accept->path is the accepted
 *   chain, bonus_token the drawn token, argmax[] is left 0.  The step is
 *   pending for dv_kv_commit like a greedy one.
 * Errors: DV_EINVAL (as dv_verify_step, plus temperature, draft_probs,
 * uniforms), DV_ECAPACITY, DV_EHIP. */
int dv_verify_step_sampled(dv_handle *h, const int32_t *tokens, const int32_t *tree_parents,
                           int32_t n_tree, dv_kv *kv, const float *draft_probs, float temperature,
                           const float *u_accept, const float *u_bonus, float *out_logits,
                           dv_accept *out_accept);

/* The sampling rule of dv_verify_step_sampled alone, on caller logits:
 * logits is device [n_tree][vocab] fp32, 16-byte aligned (row i = the
 * logits after node i).
 * Does not touch any cache and leaves no pending step (base_len is set to
 * -1).  Synchronises the handle's stream.  Errors: DV_EINVAL, DV_EHIP. */
int dv_accept_sampled(dv_handle *h, const float *logits, const int32_t *tokens,
                      const int32_t *tree_parents, int32_t n_tree, const float *draft_probs,
                      float temperature, const float *u_accept, const float *u_bonus,
                      dv_accept *out_accept);

/* The sampling rule of dv_accept_sampled without a handle and without any
 * allocation, for callers that cannot allocate device memory (serving loops
 * and harnesses that forbid hipMalloc).  Its workspace (the result struct and
 * two distribution rows) is a fixed device array of the library, 2 MiB + 1 KiB,
 * one per GPU (the current device), held until the process ends; the call
 * makes no hipMalloc/hipFree and no allocating library call.  Calls that
 * overlap on one GPU (other threads, other streams) share that array and
 * race; calls in sequence are safe (nothing in it needs to start at zero).
 *   logits: device [n_tree][vocab] fp32, 16-byte aligned;
 *   vocab: multiple of 4, 4 <= vocab <= DV_NOALLOC_MAX_VOCAB (DV_EINVAL
 *       beyond the limit, before anything is launched);
 *   stream: hipStream_t the kernel and the result copy run on (NULL =
 *       default stream); the call synchronises it;
 *   other arguments, the rule and out_accept as dv_accept_sampled.
 * Errors (message via dv_last_error(NULL)): DV_EINVAL, DV_EHIP. */
#define DV_NOALLOC_MAX_VOCAB 262144
int dv_accept_sampled_noalloc(const float *logits, const int32_t *tokens, const int32_t *tree_parents,
                              int32_t n_tree, int32_t vocab, const float *draft_probs, float temperature,
                              const float *u_accept, const float *u_bonus, void *stream,
                              dv_accept *out_accept);

/* ---- Draft side (Section 3.1 tree construction, Section 3.2 Dynamic Gated
 * Fusion, Section 3.3 multiple blocks) ---------------------------------- */

/* DGF weights, device bf16, row-major [out][in]:
 *   w_hidden [d_model][d_model], w_embed [d_model][d_model],
 *   w_gate [d_model][2 d_model] (applied to [h1 || h2]).
 * Fusion: h1 = w_hidden f, h2 = w_embed e, g = sigmoid(w_gate [h1 || h2]),
 * x0 = g h1 + (1 - g) h2 (no biases). */
typedef struct dv_dgf_weights {
    const void *w_hidden;
    const void *w_embed;
    const void *w_gate;
} dv_dgf_weights;

/* A draft handle: the draft's M blocks as a dv_config / dv_weights pair
 * (n_layers = M, weight_dtype DV_BF16; embed and lm_head are normally the
 * target's, final_norm the draft's own) plus the DGF weights.  Its KV cache
 * (dv_kv of the same shape rules) holds the draft's committed context; tree
 * nodes are written to slots [len, len + n) and never committed here.
 * Errors: as dv_verify_init, DV_EINVAL for a non-bf16 config or null DGF
 * weights. */
int dv_draft_init(const dv_config *cfg, const dv_weights *w, const dv_dgf_weights *dgf, void *stream,
                  dv_handle **out);

/* One draft pass over an n_tree-node tree (tokens / tree_parents as for
 * dv_verify_step): node i's input is DGF(feat_in[i], E[tokens[i]]), the
 * stack runs with the tree mask and positions of the verify step, and
 *   feat_out:   device [n_tree][d_model] fp32, the residual stream after the
 *               last block (the feature node i's children take as input);
 *   out_logits: device [n_tree][vocab] fp32 (after the final norm and
 *               lm_head).
 * feat_in: device [n_tree][d_model] fp32.  All device buffers 16-byte
 * aligned.  Synchronises the stream.  Errors: DV_EINVAL, DV_ESTATE (not a
 * draft handle), DV_ECAPACITY, DV_EHIP. */
int dv_draft_forward(dv_handle *h, const int32_t *tokens, const int32_t *tree_parents, int32_t n_tree,
                     dv_kv *kv, const float *feat_in, float *feat_out, float *out_logits);

/* Draft-tree construction (Section 3.1): the score of a node is the product
 * of the draft probabilities along its root path; for `depth` rounds the
 * `width` best-scoring nodes of the newest layer are expanded by their
 * `width` most probable tokens (lower id first on ties); then the root and
 * the n_tree - 1 best other nodes (earlier-created first on ties) form the
 * tree, in creation order.  Node 0 is root_token, fed root_feature (device
 * [d_model] fp32: the hidden state handed over with the accepted tokens).
 * Nodes that can no longer reach the final selection are dropped after every
 * round, so every draft pass covers at most n_tree nodes.
 * out_tokens / out_parents (host, n_tree entries) receive a tree ready for
 * dv_verify_step (entries past the returned size are -1); out_scores (host,
 * nullable) the scores.  Returns the tree size (>= 1), or a negative error:
 * DV_EINVAL (width > 16, n_tree > max_tree, bad root), DV_ESTATE,
 * DV_ECAPACITY (len + n_tree beyond the cache), DV_EHIP. */
int dv_draft_tree(dv_handle *h, int32_t root_token, const float *root_feature, dv_kv *kv, int32_t depth,
                  int32_t width, int32_t n_tree, int32_t *out_tokens, int32_t *out_parents, float *out_scores);

/* Commit the accepted path of the pending step: for k < accept_len the
 * entries of node path[k] move to slot len + k (all layers, heads, K and V;
 * all sources are read before any destination is written), then
 * kv->len += accept_len.  accept must come from the last dv_verify_step on
 * this handle and kv (same n_tree and base_len), with path a root-to-node
 * chain of that step's tree.  Errors: DV_EINVAL, DV_ESTATE, DV_EHIP. */
int dv_kv_commit(dv_handle *h, dv_kv *kv, const dv_accept *accept);

/* Build the cache from a prompt (the target's prefill before the first
 * draft round, Section 3.1; the Limitations section names long-context
 * prefill as the method's bottleneck): appends the K/V of tokens[0..n) after the kv->len
 * committed entries and commits all of them (kv->len += n).  With bf16
 * weights and n > max_tree the prompt runs as causal chunks of up to 1024
 * tokens (an MFMA GEMM with fused epilogues for the projections, a causal
 * attention kernel);
 * otherwise as chains of at most max_tree tokens through the verify step's
 * kernels.  out_next_token (host, nullable) receives the argmax after the
 * last prompt token, the root of the first draft tree.  Synchronises the
 * stream.  Errors: DV_EINVAL, DV_ECAPACITY, DV_EHIP. */
int dv_prefill(dv_handle *h, const int32_t *tokens, int32_t n, dv_kv *kv,
               int32_t *out_next_token);

/* Release the handle and its workspace (NULL is ignored). */
void dv_verify_free(dv_handle *h);

/* Message for the most recent failure on h (or of the last failed init when
 * h is NULL).  Valid until the next call on the same handle. */
const char *dv_last_error(const dv_handle *h);

/* Host-only tree preprocessing used by dv_verify_step: validates parents
 * (tree contract above, 1 <= n_tree <= 64) and writes, per node, its
 * position base_len + depth - 1, its depth (root 1) and its ancestor-or-self
 * bitmask (bit j set iff node j is on the root path of node i).  Output
 * pointers are host arrays of n_tree entries.  Returns DV_OK or DV_EINVAL. */
int dv_tree_prepare(const int32_t *tree_parents, int32_t n_tree, int32_t base_len,
                    int32_t *out_pos, int32_t *out_depth, uint64_t *out_anc);

/* Per-kernel timing with HIP events on the handle's stream.  class_mask
 * selects kernel classes (bit c for class c; 0 turns timing off); each launch
 * of a selected class is bracketed by events, read back when a step or
 * prefill synchronises.  dv_profile_read returns the summed duration (ms) and
 * launch count of one class since the last reset, and resets when
 * reset != 0.  Classes: DV_K_GEMM (weight-streaming projections and
 * lm_head), DV_K_ATTN (tree attention incl. split merge), DV_K_NORM,
 * DV_K_OTHER (argmax reduce + acceptance).  Errors: DV_EINVAL. */
#define DV_K_GEMM 0
#define DV_K_ATTN 1
#define DV_K_NORM 2
#define DV_K_OTHER 3
#define DV_K_COUNT 4
int dv_profile_enable(dv_handle *h, int32_t class_mask);
int dv_profile_read(dv_handle *h, int32_t kernel_class, double *total_ms, int64_t *launches,
                    int32_t reset);

#ifdef __cplusplus
}
#endif
#endif /* DV_H */
