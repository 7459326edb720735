/*
 * ssdref — plain CPU oracle for the tree-verification hot path of staged
 * speculative decoding (Spector & Re, "Accelerating LLM Inference with Staged
 * Speculative Decoding", arXiv 2308.04623).
 *
 * TEST INFRASTRUCTURE ONLY.  This library exists so that tests, the smoke
 * check and the benchmark's CPU-baseline leg can compare the GPU library
 * against a slow, obviously correct reference.  No product code path may
 * call it.  It shares no source, header, table or helper with the GPU
 * library.
 *
 * Arithmetic: activations, dot products, softmax and LayerNorm in fp64.
 * Stored parameters and K/V are read as their exact stored values (float32,
 * or bfloat16 bit patterns widened exactly).  K and V are rounded to the
 * storage type when produced (round-to-nearest-even), because those rounded
 * values are what every later node and later step reads from the cache.
 * Logits are rounded to float32 at the end.
 *
 * Every element is computed by one thread with a fixed summation order
 * (ascending index), so results are bitwise independent of the OpenMP thread
 * count, of the number of tree nodes and of a node's slot in the tree.
 *
 * Paper passages followed:
 *  - Sec. 2.1 (autoregressive inference): prefill builds the KV cache; each
 *    decode step feeds one token and reads the cache.
 *  - Sec. 3.1 (tree-structured batches): attention of a batch node is split
 *    into attention over the KV cache plus attention within the batch, masked
 *    by the tree; positional embeddings are set per node; the batch K/V is
 *    kept apart and the accepted slices are appended to the cache after
 *    sampling.
 *  - Sec. 2.3 (speculative decoding): draft tokens are checked in one batch;
 *    everything after the first rejection is dropped; rejection sampling
 *    keeps the oracle model's distribution.
 *
 * All pointers are host memory.  Functions return 0 on success and a
 * negative code on invalid input (nothing is written in that case).
 */
#ifndef SSDREF_H
#define SSDREF_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SSDREF_OK 0
#define SSDREF_E_ARG (-1)
#define SSDREF_E_TREE (-2)
#define SSDREF_E_CAPACITY (-3)

/* Storage type of every parameter and of the K/V cache. */
#define SSDREF_F32 0
#define SSDREF_BF16 1

#define SSDREF_ACCEPT_GREEDY 0
#define SSDREF_ACCEPT_SAMPLE_WOR 1 /* siblings were drawn without replacement */
#define SSDREF_ACCEPT_SAMPLE_IID 2 /* siblings were drawn independently      */
#define SSDREF_ACCEPT_SAMPLE_DET 3 /* siblings were chosen, not drawn (e.g. the draft's top tokens) */
#define SSDREF_ACCEPT_SAMPLE_CDF 4 /* uniforms drawn first, one per node; inverse-CDF coupling */

typedef struct {
  int32_t n_layer, d_model, n_head, d_mlp, vocab, n_pos;
  int32_t dtype; /* SSDREF_F32 or SSDREF_BF16 */
  double ln_eps;
} ssdref_config;

/* 8-bit weights (Sec. 4 lists 8-bit weights among the further speed-ups
 * and fixes no format; this is the reading taken here): symmetric, one
 * float32 scale per output row.  For row o of a bfloat16 matrix let
 * a = max_k |w[o][k]| (exact in float32).  The codes are decided in float32,
 * each operation rounded once to nearest even:
 *   r = 127 / a,   code[o][k] = clamp(rint(w[o][k] * r), -127, 127),
 *   scale[o] = a / 127;
 * a row with a < 2^-100 (zeros included) gets scale 0 and codes 0.  The model
 * then uses the weight scale[o] * code[o][k], read exactly in fp64.
 * Returns SSDREF_E_ARG (writing nothing) on a NaN or infinite weight. */
int ssdref_quantize_q8(const uint16_t *w, int32_t rows, int32_t cols, int8_t *codes, float *scales);

/* The 8-bit matrices of a bfloat16 model, from ssdref_quantize_q8: the four
 * per-layer weight matrices (arrays of n_layer pointers) and the LM head's
 * own copy of wte (wte itself stays the embedding table). */
typedef struct {
  const int8_t *const *qkv_code, *const *o_code, *const *fc_code, *const *pr_code; /* [out][in] */
  const float *const *qkv_scale, *const *o_scale, *const *fc_scale, *const *pr_scale; /* [out] */
  const int8_t *head_code;  /* [vocab][d] */
  const float *head_scale;  /* [vocab]    */
} ssdref_q8;

/* GPT-2 parameters.  Matrices are [out][in] row-major; element type per
 * config.dtype (bf16 = uint16 bit pattern).  Per-layer entries are arrays of
 * n_layer pointers.  The LM head is tied to wte.  q8 is NULL, or (bf16
 * models only) the 8-bit copies the weight matrices and the LM head are read
 * from instead of w_qkv, w_o, w_fc, w_pr and wte. */
typedef struct {
  const void *wte;   /* [vocab][d]  */
  const void *wpe;   /* [n_pos][d]  */
  const void *lnf_g; /* [d]         */
  const void *lnf_b; /* [d]         */
  const void *const *ln1_g, *const *ln1_b; /* [d]              */
  const void *const *w_qkv, *const *b_qkv; /* [3d][d], [3d]    */
  const void *const *w_o, *const *b_o;     /* [d][d], [d]      */
  const void *const *ln2_g, *const *ln2_b; /* [d]              */
  const void *const *w_fc, *const *b_fc;   /* [d_mlp][d], [d_mlp] */
  const void *const *w_pr, *const *b_pr;   /* [d][d_mlp], [d]  */
  const ssdref_q8 *q8;
} ssdref_weights;

/* Tree bookkeeping (Sec. 3.1).  parent_idx[0] must be -1 and
 * 0 <= parent_idx[i] < i for i > 0 (topological order).  Writes
 * depth[n] (root depth 0) and anc[n*n] with anc[i*n+j] = 1 iff j is i or an
 * ancestor of i.  Either output may be NULL.  Returns SSDREF_E_TREE on a
 * malformed tree. */
int ssdref_tree_info(const int32_t *parent_idx, int32_t n, int32_t *depth, uint8_t *anc);

/* Tree verification pass (Sec. 3.1).
 *  k_cache, v_cache: [n_layer][n_head][max_ctx][head_dim], rows 0..prefix_len-1 hold the prefix.
 *  k_tree, v_tree:   [n_layer][n_head][max_nodes][head_dim], written for rows 0..n_nodes-1.
 *  Node i sits at position prefix_len + depth(i) and attends to the prefix_len
 *  cached keys followed by its ancestors root..parent and itself.
 *  logits: [n_nodes][vocab] float32.
 *  n_threads <= 0 uses the OpenMP default. */
int ssdref_tree_verify(const ssdref_config *cfg, const ssdref_weights *w,
                       const void *k_cache, const void *v_cache, int32_t max_ctx, int32_t prefix_len,
                       const int32_t *tokens, const int32_t *parent_idx, int32_t n_nodes,
                       void *k_tree, void *v_tree, int32_t max_nodes,
                       float *logits, int32_t n_threads);

/* Appends the accepted nodes' K/V (path[0..path_len-1], root first) to the
 * cache at rows prefix_len..prefix_len+path_len-1 (Sec. 3.1, last sentence). */
int ssdref_kv_commit(const ssdref_config *cfg, void *k_cache, void *v_cache, int32_t max_ctx,
                     int32_t prefix_len, const void *k_tree, const void *v_tree, int32_t max_nodes,
                     const int32_t *path, int32_t path_len);

/* Accept/reject walk over the verified tree (Sec. 2.3 and 3.1).
 *  mode GREEDY: draft_probs may be NULL; temperature and seed are ignored.
 *  mode SAMPLE_*: draft_probs[u][v] is the distribution node u's children
 *  were drawn from; the target at node u is softmax(logits[u] / temperature).
 * Outputs: path[0..*path_len-1] (root first, path[0] = 0) and the one extra
 * token (bonus or corrected) in *next_token. */
int ssdref_tree_accept(int32_t mode, const int32_t *tokens, const int32_t *parent_idx, int32_t n_nodes,
                       int32_t vocab, const float *draft_probs, const float *logits, double temperature,
                       uint64_t seed, int32_t *path, int32_t *path_len, int32_t *next_token);

/* The same walk with two sampling variants (Sec. 4 evaluates top-k sampling
 * with k = 50, T = 1):
 *  top_k > 0: the target at node u is softmax(logits[u] / temperature) over
 *    the top_k largest logits of the row only (ties at the cut go to the
 *    lower token id), zero elsewhere; top_k = 0 keeps the whole vocabulary.
 *    Greedy acceptance ignores it.
 *  mode SAMPLE_DET: the children of a node were chosen deterministically
 *    (draft_probs must be NULL): each child in turn is accepted with
 *    probability r(x) / Z (the residual target mass at its token); on
 *    rejection that token's mass is removed.  The extra token is drawn from
 *    the residual, as in the other sampling modes.
 *  mode SAMPLE_CDF (Sec. 4 suggests drawing the multinomial CDF samples
 *    first and assembling the batch around them; draft_probs must be NULL):
 *    node u's uniform is U_u = ssdref_uniform(seed, 2, u), known before the
 *    tree is built.  At node u the oracle's token is x = the smallest id
 *    whose running target sum (ascending id, fp64) exceeds U_u (if rounding
 *    leaves none, the last id with positive target).  The walk moves to the
 *    first child (lowest index) whose token is x; when none is, x is the
 *    extra token.  Every emitted token is then an exact draw from the
 *    target given the tokens before it, whatever tree was assembled. */
int ssdref_tree_accept_k(int32_t mode, const int32_t *tokens, const int32_t *parent_idx, int32_t n_nodes,
                         int32_t vocab, const float *draft_probs, const float *logits, double temperature,
                         int32_t top_k, uint64_t seed, int32_t *path, int32_t *path_len, int32_t *next_token);

/* The token drawn from softmax(row / temperature) (whole vocabulary, fp64)
 * at uniform U by inverse CDF in ascending token id: the oracle's token of
 * SAMPLE_CDF at a node, here at a given uniform (CDF-first tree assembly
 * picks the draft's tokens this way).  Returns -1 on invalid input. */
int32_t ssdref_cdf_pick(const float *row, int32_t vocab, double temperature, double U);

/* Philox4x64-10 (Salmon, Moraes, Dror, Shaw, SC'11): out = bijection(ctr; key). */
void ssdref_philox4x64_10(const uint64_t key[2], const uint64_t ctr[4], uint64_t out[4]);

/* Uniform double in [0,1): top 53 bits of word 0 of Philox4x64-10 with
 * key (seed, stream) and counter (n, 0, 0, 0). */
double ssdref_uniform(uint64_t seed, uint64_t stream, uint64_t n);

/* float32 -> bfloat16 and fp64 -> bfloat16, round-to-nearest-even. */
uint16_t ssdref_round_bf16(double x);

#ifdef __cplusplus
}
#endif
#endif
