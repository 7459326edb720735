/*
 * ssd.h — C ABI of libssd, the MI355X (gfx950) tree-verification library for
 * staged speculative decoding (Spector & Re, arXiv 2308.04623).
 *
 * One decoding step of the paper's method, on one GPU:
 *   ssd_tree_verify  scores every node of a speculative token tree against the
 *                    KV cache of the accepted prefix in one decoder pass
 *                    (Sec. 3.1: attention split into attention over the cache
 *                    plus tree-masked attention inside the batch, positions
 *                    set per node, the batch's own K/V kept apart);
 *   ssd_tree_accept  walks the tree and keeps the longest path the model
 *                    agrees with, plus one extra token (Sec. 2.3; greedy, or
 *                    rejection sampling that keeps the model's distribution);
 *   ssd_kv_commit    appends the accepted nodes' K/V to the cache (Sec. 3.1,
 *                    last step).
 *
 * Conventions shared by every call:
 *  - Device pointers are HIP device memory owned by the caller (for example
 *    torch tensors' data_ptr()); the library never frees them.  Host
 *    pointers are ordinary host memory, read before the call returns.
 *  - `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *    Work is enqueued asynchronously; no call synchronises the host except
 *    ssd_model_create (which waits for its one-time weight repacking).
 *  - Every argument, tree and capacity check runs on the host before anything
 *    is enqueued; on error nothing is enqueued and outputs are untouched.
 *    Statuses are negative on error; ssd_last_error() gives a thread-local
 *    message.  Asynchronous device faults surface as SSD_E_DEVICE later.
 *  - A handle is used by one host thread and one stream at a time.
 *
 * Model: GPT-2, pre-LayerNorm blocks, tanh GELU, learned absolute positions,
 * LM head tied to the token embedding.  All parameters and the K/V cache use
 * one storage type (float32 or bfloat16); accumulation is float32.  For
 * bfloat16 models the weight GEMMs multiply float16 operands: the weights
 * converted to float16 (exact for 0 and magnitudes in [2^-17, 65504], within
 * 2^-25 below; a weight past 65504 makes ssd_model_create fail) and the
 * activations rounded to float16 (an activation past 65504 is counted in the
 * session's error counter, see ssd_kv_error_count).
 */
#ifndef SSD_H
#define SSD_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  SSD_OK = 0,
  SSD_E_INVALID_ARG = -1,  /* null pointer, bad size, bad config, bad token id  */
  SSD_E_INVALID_TREE = -2, /* parent_idx[0] != -1 or parent_idx[i] not in [0,i)  */
  SSD_E_CAPACITY = -3,     /* more nodes / context / positions than allocated     */
  SSD_E_DEVICE = -4,       /* a HIP runtime call failed                           */
  SSD_E_UNSUPPORTED = -5   /* shape the kernels do not handle (see ssd_model_create) */
} ssd_status;

typedef enum { SSD_F32 = 0, SSD_BF16 = 1 } ssd_dtype;

typedef enum {
  SSD_ACCEPT_GREEDY = 0,     /* argmax walk                                          */
  SSD_ACCEPT_SAMPLE_WOR = 1, /* rejection sampling; siblings were drawn without replacement */
  SSD_ACCEPT_SAMPLE_IID = 2, /* rejection sampling; siblings were drawn independently       */
  SSD_ACCEPT_SAMPLE_DET = 3, /* rejection sampling; siblings were chosen (e.g. the draft's top
                                tokens), each proposed with certainty: no draft rows      */
  SSD_ACCEPT_SAMPLE_CDF = 4  /* CDF-first: one uniform per node, drawn before the tree is
                                built; the oracle's token by inverse CDF (no draft rows)   */
} ssd_accept_mode;

typedef struct {
  int32_t n_layer, d_model, n_head, d_mlp, vocab, n_pos;
  ssd_dtype dtype; /* storage type of every parameter and of the K/V cache */
  float ln_eps;    /* LayerNorm epsilon (GPT-2: 1e-5) */
} ssd_config;

/* Device pointers to the parameters, caller-owned, in the config's storage
 * type.  Matrices are [out][in] row-major; per-layer entries are HOST arrays
 * of n_layer device pointers.  Must stay valid until ssd_model_destroy. */
typedef struct {
  const void *wte;   /* [vocab][d_model]: token embedding and tied LM head */
  const void *wpe;   /* [n_pos][d_model]                                   */
  const void *lnf_g; /* [d_model]                                          */
  const void *lnf_b; /* [d_model]                                          */
  const void *const *ln1_g, *const *ln1_b; /* [d_model]                           */
  const void *const *w_qkv, *const *b_qkv; /* [3 d_model][d_model], [3 d_model]   */
  const void *const *w_o, *const *b_o;     /* [d_model][d_model], [d_model]       */
  const void *const *ln2_g, *const *ln2_b; /* [d_model]                           */
  const void *const *w_fc, *const *b_fc;   /* [d_mlp][d_model], [d_mlp]           */
  const void *const *w_pr, *const *b_pr;   /* [d_model][d_mlp], [d_model]         */
} ssd_weights;

typedef struct ssd_model ssd_model; /* opaque */
typedef struct ssd_kv ssd_kv;       /* opaque: one decoding session's cache + workspaces */
typedef struct ssd_graph ssd_graph; /* opaque: a captured verification pass */

/* A token tree in host memory (Sec. 3.1).  Node 0 is the root: the last
 * emitted token, not yet in the cache.  parent_idx[0] = -1 and
 * 0 <= parent_idx[i] < i (topological order). */
typedef struct {
  const int32_t *tokens;     /* [n_nodes] */
  const int32_t *parent_idx; /* [n_nodes] */
  int32_t n_nodes;
  int32_t vocab;
  ssd_accept_mode mode;
  float temperature; /* sampling modes: target = softmax(logits / temperature) */
  int32_t top_k;     /* sampling modes: > 0 restricts the target to the row's top_k
                        largest logits (ties at the cut to the lower token id,
                        renormalised; Sec. 4 uses k = 50, T = 1); 0 = whole vocabulary */
} ssd_tree;

/* Loads a model.  Supported shapes: d_model % 32 == 0, d_mlp % 32 == 0,
 * head_dim (= d_model / n_head) of 32 or 64.  For bfloat16 the library
 * repacks every matrix (and the LM head) once into a private copy laid out in
 * matrix-core tile order (freed by ssd_model_destroy); this call waits for it.
 * Errors: SSD_E_INVALID_ARG, SSD_E_UNSUPPORTED (also: a bfloat16 matrix or
 * LM-head weight of magnitude above 65504, or NaN, which its float16 copy
 * cannot hold), SSD_E_DEVICE. */
ssd_status ssd_model_create(const ssd_config *cfg, const ssd_weights *w, void *stream, ssd_model **out);

/* Loads a bfloat16 model with 8-bit weights (Sec. 4 names 8-bit weights
 * among the further speed-ups; the format is this library's reading): the
 * four weight matrices of every layer and the tied LM head are replaced by
 * symmetric 8-bit codes with one float32 scale per output row, made once
 * here from the bfloat16 weights in w.  Per row, with a the largest weight
 * magnitude, the codes are decided in float32 with every operation rounded
 * to nearest even: r = 127 / a, code = clamp(rint(w * r), -127, 127),
 * scale = a / 127 (rows with a < 2^-100: scale 0, codes 0).  The model then
 * multiplies scale * code, half the weight bytes of ssd_model_create's
 * float16 copies; the embedding lookups, biases and LayerNorm parameters
 * stay bfloat16.  This is a different model from the bfloat16 one: its
 * logits follow the 8-bit weights.  The K/V cache stays bfloat16.  Extra
 * requirements: dtype SSD_BF16, d_model and d_mlp multiples of 64.  Errors:
 * as ssd_model_create; SSD_E_UNSUPPORTED also for a NaN or infinite weight. */
ssd_status ssd_model_create_q8(const ssd_config *cfg, const ssd_weights *w, void *stream, ssd_model **out);
void ssd_model_destroy(ssd_model *m);

/* Draft view for staged speculation (Sec. 3.2: a cheaper model proposes the
 * tokens the oracle checks; here the oracle's first n_layer blocks followed
 * by its final LayerNorm and tied LM head).  The view shares every device
 * buffer with m (weights, packed copies), allocates nothing on the device,
 * and must be destroyed (ssd_model_destroy, which frees only the view)
 * before m.  Its layers' K/V are the oracle's, so a draft session may bind
 * the oracle's cache: layer l of the view is layer l of the
 * [n_layer][n_head][rows][head_dim] buffers.  1 <= n_layer <= m's layers.
 * Errors: SSD_E_INVALID_ARG. */
ssd_status ssd_model_prefix_view(const ssd_model *m, int32_t n_layer, ssd_model **out);

/* Bytes the caller must allocate for the cache (each of K and V:
 * [n_layer][n_head][max_ctx][head_dim]) and the tree scratch (each of K and V:
 * [n_layer][n_head][max_nodes][head_dim]) in the storage type. */
ssd_status ssd_kv_bytes(const ssd_config *cfg, int32_t max_ctx, int32_t max_nodes, size_t *cache_bytes,
                        size_t *tree_bytes);

/* Binds caller-owned K/V buffers to a session and allocates the session's
 * workspaces (activations, attention partials, accept scratch, pinned
 * staging).  max_nodes <= 1024.  Errors: SSD_E_INVALID_ARG, SSD_E_CAPACITY,
 * SSD_E_DEVICE. */
ssd_status ssd_kv_create(const ssd_model *m, int32_t max_ctx, int32_t max_nodes, void *k_cache, void *v_cache,
                         void *k_tree, void *v_tree, ssd_kv **out);
void ssd_kv_destroy(ssd_kv *kv);

/* Tree verification pass (Sec. 3.1).  Node i sits at position
 * prefix_len + depth(i) and attends to cache rows 0..prefix_len-1, then to
 * its ancestors root..parent and itself in the tree scratch.  Writes every
 * node's K/V to the tree scratch rows 0..n_nodes-1 and
 * logits[n_nodes][vocab] (float32, device).  Never modifies the cache, so
 * repeating a call gives the same result.
 * Errors: SSD_E_INVALID_ARG (null, token out of range), SSD_E_INVALID_TREE,
 * SSD_E_CAPACITY (n_nodes > max_nodes, prefix_len > max_ctx,
 * prefix_len + max depth >= n_pos), SSD_E_DEVICE. */
ssd_status ssd_tree_verify(const ssd_model *m, ssd_kv *kv, int32_t prefix_len, const int32_t *tree_tokens,
                           const int32_t *parent_idx, int32_t n_nodes, float *logits, void *stream);

/* ssd_tree_verify followed by the greedy accept walk of ssd_tree_accept
 * (SSD_ACCEPT_GREEDY) on the logits it wrote, with the same outputs as that
 * pair of calls, bit for bit.  When the pass runs as the persistent single
 * launch (see ssd_options), its LM head also leaves each workgroup's largest
 * logit and token per node, so the walk needs no second read of the
 * [n_nodes][vocab] logits (Sec. 4, greedy "deterministic" decoding).
 * Errors: as ssd_tree_verify, plus SSD_E_INVALID_ARG for a null output. */
ssd_status ssd_tree_verify_greedy(const ssd_model *m, ssd_kv *kv, int32_t prefix_len, const int32_t *tree_tokens,
                                  const int32_t *parent_idx, int32_t n_nodes, float *logits, int32_t *accepted_path,
                                  int32_t *path_len, int32_t *next_token, void *stream);

/* The verification pass from layer start_layer on, for a tree whose first
 * layers a draft already ran.  The paper does not describe this (its draft,
 * Sec. 3.2 and 4, is a separate small model): it applies when the draft is
 * ssd_model_prefix_view of this model, whose layers are this model's first
 * ones, so their outputs for a node are the oracle's.  x_in ([n_nodes][d_model] fp32,
 * device) is every node's residual stream at the input of start_layer, and
 * the session's tree scratch rows 0..n_nodes-1 must already hold the nodes'
 * K/V of layers 0..start_layer-1 (ssd_tree_reuse provides both).  Layers
 * start_layer.. then run exactly as in ssd_tree_verify, which a pass from
 * layer 0 is.  With accepted_path, path_len and next_token all set, the
 * greedy walk of ssd_tree_verify_greedy follows; all NULL, none.  Errors:
 * as ssd_tree_verify, plus SSD_E_INVALID_ARG for start_layer outside
 * [0, n_layer), a NULL x_in with start_layer > 0, or greedy outputs only
 * partly set. */
ssd_status ssd_tree_verify_from(const ssd_model *m, ssd_kv *kv, int32_t prefix_len, const int32_t *tree_tokens,
                                const int32_t *parent_idx, int32_t n_nodes, int32_t start_layer, const float *x_in,
                                float *logits, int32_t *accepted_path, int32_t *path_len, int32_t *next_token,
                                void *stream);

/* Hands a draft pass's work to the oracle's session for ssd_tree_verify_from:
 * for i < n, the tree K/V rows at src's tree scratch row src_rows[i] of
 * every layer that src's last pass ran (the last ssd_tree_verify,
 * ssd_tree_verify_greedy, ssd_tree_verify_from or graph launch on src) go
 * to dst's tree scratch row i, and the residual stream that pass left for
 * node src_rows[i] (after its last layer) goes to x_out[i] ([n][d_model]
 * fp32, device); ssd_tree_verify_from then starts at that layer count.
 * The model of that pass must be a layer prefix of dst's
 * (ssd_model_prefix_view), and the two sessions' tree scratch buffers must
 * not overlap.  Enqueue on the stream of that pass, after it.
 * 1 <= n <= min(256, dst's max_nodes); src_rows is a HOST array, each
 * below the node count of src's last pass.  Errors: SSD_E_INVALID_ARG
 * (null, src == dst, shapes, no pass yet, a row outside the last pass),
 * SSD_E_CAPACITY, SSD_E_DEVICE. */
ssd_status ssd_tree_reuse(const ssd_kv *src, ssd_kv *dst, int32_t n, const int32_t *src_rows, float *x_out,
                          void *stream);

/* Accept/reject walk (Sec. 2.3, 3.1) over logits from ssd_tree_verify.
 *  greedy: a node is kept when its parent is kept and its token is the
 *    parent's argmax (lowest token id on ties); the deepest kept node (lowest
 *    index on ties) ends the path and its argmax is the extra token.
 *  sampling: recursive rejection sampling down the tree.  For the two
 *    drawn modes draft_probs ([n_nodes][vocab], device) row u is the
 *    distribution node u's children were drawn from: child x is accepted
 *    with probability min(1, r(x) / q(x)) (r the residual target, q the
 *    draft row, in the without-replacement mode with the rejected tokens'
 *    draft mass removed); on rejection r becomes max(r - q, 0).  In the
 *    chosen mode (SSD_ACCEPT_SAMPLE_DET, draft_probs NULL) child x is
 *    accepted with probability r(x) and on rejection x's mass leaves r.  If
 *    no child of the last accepted node is accepted, the extra token is
 *    drawn from the residual (the full target at a leaf).  Uniforms come
 *    from Philox4x64-10 keyed by (rng_seed, 0) with counter
 *    (child index, 0, 0, 0) for the test of that child, and (rng_seed, 1)
 *    with counter (last node) for the extra token.
 *  CDF-first (SSD_ACCEPT_SAMPLE_CDF, draft_probs NULL; Sec. 4 suggests
 *    drawing the multinomial CDF samples first and assembling the batch
 *    around them): node u's uniform U_u comes from key (rng_seed, 2),
 *    counter (u, 0, 0, 0) (ssd_uniform gives it on the host, before the
 *    tree is built).  The oracle's token at u is the smallest token id whose
 *    running target sum (ascending id) exceeds U_u; the walk moves to the
 *    first child (lowest index) carrying it, and where none does it is the
 *    extra token.  Each emitted token is an exact draw from the target given
 *    the ones before it provided the tree obeys one rule: U_u may decide u's
 *    children, but no node's index, token or presence may depend on its own
 *    uniform or its descendants'.
 * Outputs (device): accepted_path[0..*path_len-1] root first (path[0] = 0),
 * *next_token.  Emitted tokens are tokens[path[1..]] then next_token.
 * draft_probs must be non-NULL exactly for the two drawn modes; top_k < 0 is
 * SSD_E_INVALID_ARG; a sampling mode with vocab above 131072 is
 * SSD_E_CAPACITY.  The sampling walk runs on ceil(vocab / 2048)
 * workgroups that wait for each other; if they cannot all run at once
 * within 0.5 s (the GPU held by other work), the walk gives up: *path_len
 * is set to 0 (never a valid length) and the session's error counter counts
 * it. */
ssd_status ssd_tree_accept(ssd_kv *kv, const ssd_tree *tree, const float *draft_probs, const float *oracle_logits,
                           uint64_t rng_seed, int32_t *accepted_path, int32_t *path_len, int32_t *next_token,
                           void *stream);

/* The accept walk of ssd_tree_accept (same arguments, same outputs, same
 * kernels) for callers that cannot allocate device memory: code under HIP
 * graph capture, tight serving loops, harnesses that forbid hipMalloc.  It
 * needs no session and calls no allocating routine: its scratch (the staged
 * tree, argmax partials, the sampling walk's exchange area) is one
 * file-scope device array of 209,408 bytes that every GPU the library runs on holds
 * until the process ends, and the tree reaches the device inside the kernel
 * arguments.  Limits: n_nodes <= 256 and vocab <= 65536 (SSD_E_CAPACITY
 * beyond).  All calls on one GPU share that GPU's array: calls that overlap
 * on one GPU (two streams, or two host threads) race; calls ordered on one
 * stream do not.  A sampling walk that gives up sets *path_len = 0 (there
 * is no session to count it).  Errors: as ssd_tree_accept, plus
 * SSD_E_CAPACITY. */
ssd_status ssd_tree_accept_noalloc(const ssd_tree *tree, const float *draft_probs, const float *oracle_logits,
                                   uint64_t rng_seed, int32_t *accepted_path, int32_t *path_len,
                                   int32_t *next_token, void *stream);

/* Appends tree scratch rows accepted_path[0..*path_len-1] (device arrays, as
 * written by ssd_tree_accept) to cache rows prefix_len.. (Sec. 3.1).  Reads
 * the path on the device, so no host sync is needed between accept and
 * commit.  Rows that would fall past max_ctx, or path entries outside
 * [0, max_nodes), are skipped and counted in the session's error counter. */
ssd_status ssd_kv_commit(ssd_kv *kv, int32_t prefix_len, const int32_t *accepted_path, const int32_t *path_len,
                         void *stream);

/* The session's error counter since it began (synchronises the stream): it
 * counts commit rows skipped as out of range, persistent verification passes
 * that ended early (a bounded wait timed out, or the launch did not get one
 * workgroup per CU; that pass's logits are undefined) and GEMM inputs that
 * overflowed float16 (see ssd_tree_verify).  A caller that needs a valid
 * result checks that it did not grow. */
ssd_status ssd_kv_error_count(ssd_kv *kv, void *stream, uint32_t *count);

/* Top-k of every row of logits[n_rows][vocab] (vocab of kv's model), for
 * building draft trees (Sec. 3.1, 3.2: candidate continuations of a node are
 * the draft's most likely tokens).  Writes, on the device, idx[n_rows][k]
 * (token ids, decreasing logit, lower id first on ties), val[n_rows][k]
 * (their logits) and, if lse is not NULL, lse[n_rows] = log sum exp of the
 * row (so that val - lse is the log-probability).  Uses kv's workspace, so
 * calls on one session are ordered by the stream.  1 <= k <= 8,
 * 1 <= n_rows <= max_nodes.  Errors: SSD_E_INVALID_ARG, SSD_E_CAPACITY,
 * SSD_E_DEVICE. */
ssd_status ssd_topk(ssd_kv *kv, const float *logits, int32_t n_rows, int32_t k, int32_t *idx, float *val, float *lse,
                    void *stream);

/* Captures one verification pass (same arguments as ssd_tree_verify) into a
 * HIP graph; ssd_graph_launch replays it on the given stream with the same
 * tree and prefix.  Capture runs on a library-private stream (nothing
 * executes during capture; `stream` is unused).  Used to run the pass
 * without per-kernel host launch overhead. */
ssd_status ssd_graph_capture_verify(const ssd_model *m, ssd_kv *kv, int32_t prefix_len, const int32_t *tree_tokens,
                                    const int32_t *parent_idx, int32_t n_nodes, float *logits, void *stream,
                                    ssd_graph **out);
/* The same for ssd_tree_verify_greedy: the graph replays the pass and the
 * greedy walk into the given device outputs. */
ssd_status ssd_graph_capture_verify_greedy(const ssd_model *m, ssd_kv *kv, int32_t prefix_len,
                                           const int32_t *tree_tokens, const int32_t *parent_idx, int32_t n_nodes,
                                           float *logits, int32_t *accepted_path, int32_t *path_len,
                                           int32_t *next_token, void *stream, ssd_graph **out);
ssd_status ssd_graph_launch(ssd_graph *g, void *stream);
void ssd_graph_destroy(ssd_graph *g);

/* Host-only tree checks (no GPU needed).  Validates topology and token ids;
 * writes the maximum depth. */
ssd_status ssd_validate_tree(const int32_t *tokens, const int32_t *parent_idx, int32_t n, int32_t vocab,
                             int32_t *max_depth);

/* Host-only tree bookkeeping as used by ssd_tree_verify: depth[n] and the
 * ancestor-or-self bitmask anc[n][ceil(n/64)] (bit j of word j/64 of row i
 * is set iff node j is node i or one of its ancestors). */
ssd_status ssd_tree_prep(const int32_t *parent_idx, int32_t n, int32_t *depth, uint64_t *anc);

/* Per-session switches (each session has its own; the defaults are 0, 0, 1).
 *   pass_mode: how a bfloat16 verification pass runs (Sec. 2.1: a decode
 *     step streams every weight once; Sec. 3.1: one step scores the whole
 *     tree).
 *     0 = automatic: the persistent single launch when the session supports
 *       it (head dimension 64, a 256-CU device with 8 XCDs) and the tree has
 *       at most 64 nodes, else one kernel per sub-layer;
 *     1 = always one kernel per sub-layer;
 *     2 = the persistent single launch only (up to 64 nodes):
 *       ssd_tree_verify and ssd_graph_capture_verify return SSD_E_UNSUPPORTED
 *       where it does not apply.
 *     The persistent launch runs every layer in one kernel: 256 workgroups
 *     (one per CU) hand results to each other through flags in device
 *     memory.  Every wait inside it is bounded; if one times out (200 ms) the
 *     launch ends early, its logits are undefined, and the session's error
 *     counter (ssd_kv_error_count) is incremented.  Both ways meet the same
 *     tolerance against the definition; their logits differ in the last bits.
 *   gemm_path: the per-sub-layer kernels' weight GEMMs, bfloat16 models
 *     only: 0 = automatic (by node count), 1 = vector ALU, 2 = matrix cores.
 *   weight_prefetch: 1 = every per-sub-layer bfloat16 pass the session
 *     enqueues (or a graph of it replays) gets a prefetcher kernel on a
 *     stream of the session's own; it follows progress signals the pass's
 *     kernels raise and loads each weight GEMM's fragments into the L2 of the
 *     XCD whose workgroups will read them, a few kernels ahead.  The pass
 *     never waits for it; it stops waiting for signals 50 ms after it starts.
 *     0 = off.  Results are bitwise the same either way.  ssd_kv_destroy
 *     waits for the session's prefetchers.
 * A captured graph keeps the pass mode and GEMM path in force when it was
 * captured.  Errors: SSD_E_INVALID_ARG (null, or a value out of range). */
typedef struct {
  int32_t pass_mode;
  int32_t gemm_path;
  int32_t weight_prefetch;
} ssd_options;

ssd_status ssd_kv_set_options(ssd_kv *kv, const ssd_options *opt);
ssd_status ssd_kv_get_options(const ssd_kv *kv, ssd_options *opt);

/* Inverse-CDF picks for CDF-first tree assembly (Sec. 4: draw the
 * multinomial CDF samples first, then assemble the batch around them): for
 * query q, tokens[q] (device) is the token drawn from
 * softmax(logits[rows[q]] / temperature) over the row's vocab entries at the
 * uniform uniforms[q], by inverse CDF in ascending token id (the order
 * SSD_ACCEPT_SAMPLE_CDF draws the oracle's tokens in).  logits:
 * [n_rows][vocab] device, vocab at most the model's; rows, uniforms: HOST
 * arrays of n_queries (1..64), read before the call returns.  Errors:
 * SSD_E_INVALID_ARG (null, vocab outside [1, the model's vocab], a row
 * outside [0, n_rows), a uniform outside [0, 1), temperature <= 0,
 * n_queries outside [1, 64]), SSD_E_CAPACITY (n_rows outside
 * [1, max_nodes]), SSD_E_DEVICE. */
ssd_status ssd_cdf_pick(ssd_kv *kv, const float *logits, int32_t n_rows, int32_t vocab, float temperature,
                        int32_t n_queries, const int32_t *rows, const double *uniforms, int32_t *tokens, void *stream);

/* The uniform ssd_tree_accept draws (Philox4x64-10 with key (seed, stream)
 * and counter (counter, 0, 0, 0); the top 53 bits of the first output word
 * times 2^-53), computed on the host.  A CDF-first tree builder
 * (SSD_ACCEPT_SAMPLE_CDF) reads node u's uniform as ssd_uniform(rng_seed, 2,
 * u) before the tree is verified.  Pure host function. */
double ssd_uniform(uint64_t seed, uint64_t stream, uint64_t counter);

const char *ssd_status_string(ssd_status s);
const char *ssd_last_error(void);

#ifdef __cplusplus
}
#endif
#endif
