// Internal declarations shared by the HIP kernels (kernels.hip) and the host
// runtime (runtime.hip) of libssd.  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <string>

namespace ssd {

// Epilogues of the skinny GEMM Y[n][o] = sum_k A[n][k] W[o][k].
enum EpiKind : int {
  EPI_QKV = 0,    // +bias; o < d -> q (fp32); d <= o < 2d -> K scratch; 2d <= o -> V scratch
  EPI_RESID = 1,  // x[n][o] += y + bias[o]
  EPI_GELU = 2,   // out[n][o] = gelu_tanh(y + bias[o])  (storage of the activation buffer)
  EPI_LOGITS = 3,  // logits[n][o] = y
  EPI_PARTIAL = 4  // part[split][n][o] = y (split-K sum of a residual GEMM, no bias)
};

// root-path entries staged per node at a fixed stride
constexpr int kPath32 = 32;

// most k-splits a residual GEMM uses
constexpr int kMaxSplits = 8;

struct Epi {
  const void* bias;  // storage type, or nullptr
  int N;             // valid nodes in this launch
  int M;             // valid output rows
  int node0;         // node offset of this launch (outputs go to node0 + n)
  // EPI_QKV
  float* q;
  void* kt;
  void* vt;
  int d, H, DH, max_nodes;
  // EPI_RESID
  float* x;
  // EPI_GELU
  void* out;
  int ldo;  // GEMM-input leading dimension: fp32 row stride, bf16 k-steps (K/32)
  // EPI_LOGITS
  float* logits;
  long long ldl;
  // EPI_PARTIAL
  float* part;
  long long part_stride;  // elements between splits
  int split;              // set by the kernel from blockIdx.y
  unsigned long long* sig;  // pass signal counter (nullptr: none)
  unsigned* err;            // session error counter: float16 GEMM inputs out of range (nullptr: none)
  const float* wscale;      // 8-bit weights: the rows' scales (nullptr: float16 weight fragments)
};

// tile shape of the bf16 GEMM for a node count: node tiles of 16, row blocks
// per workgroup, k-steps per staged chunk, nodes of the vector path
struct GemmCfg {
  int nt, rb, ck, nv, nw;  // nw: waves per workgroup
};

// launch geometry of one bf16 GEMM: block (bx, by) owns weight row blocks
// bx RB .. bx RB + RB - 1 (rows past RBtot read row block RBtot - 1 and are
// never stored) and k-steps by kcs .. by kcs + kcs - 1 (clamped to KC)
struct GemmGeom {
  int RB, kcs, gx, gy, KC, RBtot;
};

// ---- weight prefetch from a second stream
//
// Every kernel of a bfloat16 pass bumps a signal counter when it starts
// (block 0): the embedding, then per layer LN1, QKV GEMM, attention split,
// attention merge, attention-out GEMM, LN2, MLP up, MLP down.  A prefetcher
// kernel launched on another stream beside the pass waits for these signals
// and loads each weight GEMM's fragments into the L2 of the XCD that will
// read them a few kernels ahead: block b of every launch of a queue runs on
// XCD (b + c) mod 8 with one c per queue, which the embedding records.
enum SigKernel { SIG_LN1 = 0, SIG_QKV, SIG_SPLIT, SIG_MERGE, SIG_OUT, SIG_LN2, SIG_FC, SIG_PROJ, kSigPerLayer };
// counter value (past a pass's base) once kernel k of layer l has started
inline __host__ __device__ int sig_index(int l, int k) { return 2 + kSigPerLayer * l + k; }
inline int sigs_per_pass(int L) { return 1 + kSigPerLayer * L; }

struct PfGeom {
  int KC, RBtot, RB, kcs, gx, nblk;  // a GEMM launch (see GemmGeom), nblk = gx * gy
};
struct PrefetchPlan {
  const void* const* W;     // device [4][L]: packed QKV, attention-out, MLP-up, MLP-down weights
  int L;
  PfGeom geo[4];            // their launches at this pass's node count
  unsigned long long* sig;  // the session's signal counter
  const unsigned* xcc0;     // XCD of block 0 of the pass's embedding
  unsigned long long base;  // counter value before this pass
  unsigned long long timeout;  // s_memrealtime ticks (100 MHz) before the prefetcher stops waiting
  unsigned* sink;           // written only when the folded loads equal `magic` (keeps them alive)
  unsigned magic;
};

struct AttnArgs {
  const float* q;       // [N][d]
  const void* kc;       // cache, this layer: [H][max_ctx][DH]
  const void* vc;
  const void* kt;       // tree scratch, this layer: [H][max_nodes][DH]
  const void* vt;
  const int* depth;     // [N]
  const int* anc_off;   // [N] offset of node n's root path in ancl
  const int* ancl;      // root paths, root first, node itself last
  const int* path32;    // [N][kPath32]: first entries of each root path, padded with the node
  void* out;            // attention output in the GEMM-input layout
  int ldo;              // GEMM-input leading dimension (fp32: d, bf16: d / 32)
  float* part;          // fp32 models: prefix partials [H][S][N][DH + 2] (max, sum of exp, output);
                        // bf16 models: parts [H][nsplit][N] of 16 + 2 DH bytes (max and sum
                        // float32, 8 bytes of padding, output float16), one per prefix chunk
  int S;                // fp32 models: prefix tiles of 64 cache rows
  int N, P, d, H, max_ctx, max_nodes;
  float scale;
  // bf16 models
  int CL;               // cache rows per prefix chunk (attn_chunk(P, H))
  int nsplit;           // prefix chunks (attn_nsplit(P, H))
  unsigned long long* sig;  // pass signal counter (nullptr: none); both kernels signal
  unsigned* err;            // session error counter: float16 outputs out of range (nullptr: none)
};

// bf16 attention: cache rows per prefix chunk, a multiple of 32 between 64
// and kAttnMaxChunk, as few rows as keep the split kernel's H x nsplit
// blocks within one per CU (256) where the prefix allows: 64 up to
// P = 768 at 20 heads, 192 at P = 2048.  A function of the prefix length and
// the head count only, so that a node's result does not depend on the tree.
constexpr int kAttnMaxChunk = 256;
inline int attn_chunk(int P, int H) {
  const int per = 256 / H > 0 ? 256 / H : 1;  // chunks per head
  int c = (P + per - 1) / per;
  c = (c + 31) / 32 * 32;
  if (c < 64) c = 64;
  if (c > kAttnMaxChunk) c = kAttnMaxChunk;
  return c;
}
inline int attn_nsplit(int P, int H) { return P > 0 ? (P + attn_chunk(P, H) - 1) / attn_chunk(P, H) : 0; }
// most prefix chunks for any P <= max_ctx
inline int attn_max_nsplit(int max_ctx, int H) {
  int mx = 0;
  for (int P = 1; P <= max_ctx; P += (P < 8192 ? 1 : 256)) mx = attn_nsplit(P, H) > mx ? attn_nsplit(P, H) : mx;
  return attn_nsplit(max_ctx, H) > mx ? attn_nsplit(max_ctx, H) : mx;
}

// ---- launchers (kernels.hip); all enqueue on `s` and return the launch status
hipError_t launch_embed(int f32, const void* wte, const void* wpe, const int* tokens, const int* pos, int N, int d,
                        float* x, unsigned long long* sig, unsigned* xcc0, hipStream_t s);
// x += bias + part[0..S-1] (if S > 0), then LayerNorm into the GEMM-input
// buffer a (lda: fp32 row stride, or bf16 k-steps d / 32; see st_act)
hipError_t launch_ln(int f32, float* x, int N, int d, const float* part, int S, size_t pstride, const void* bias,
                     const void* g, const void* b, float eps, void* a, int lda, unsigned long long* sig,
                     unsigned* err, hipStream_t s);
hipError_t launch_gemm_f32(int kind, const float* W, int M, int K, const float* act, int lda, const Epi& ep,
                           hipStream_t s);
GemmCfg gemm_cfg(int N, int vec, int kind);
// k-steps per split and number of splits (EPI_PARTIAL only; 1 otherwise)
int gemm_split_kc(int M, int K, int N, int vec, int want_split, int* splits);
// whether a matrix-core GEMM over N nodes (of one launch) takes the
// wide-tree kernel (row blocks x node tiles per workgroup)
bool gemm_wide(int vec, int N);
GemmGeom gemm_geom(int kind, int vec, int M, int K, int N, int kcs);
// Wp: weights packed in 16x32 float16 fragments (see pack), or, with
// ep.wscale set, in 16x32 8-bit fragments (see pack_q8); act: activations of
// this launch's first node in fragment order (see st_act); kcs k-steps per
// split (grid.y = ceil(K/32 / kcs))
hipError_t launch_gemm_bf16(int kind, int vec, const void* Wp, int M, int K, const uint16_t* act, int kcs,
                            const Epi& ep, hipStream_t s);
hipError_t launch_attn(int f32, int DH, const AttnArgs& a, hipStream_t s);
hipError_t launch_prefetcher(const PrefetchPlan& pp, hipStream_t s);
// bad: device counter of packed 16-byte groups holding a weight past float16's range
hipError_t launch_pack_bf16(const uint16_t* W, int M, int K, void* out, unsigned* bad, hipStream_t s);
size_t packed_bytes(int M, int K);
// 8-bit copy of a bf16 matrix: fragments (packed_q8_bytes) and scales
// [ceil(M/16) 16] float32; bad counts rows holding a NaN or infinite weight
hipError_t launch_pack_q8(const uint16_t* W, int M, int K, void* out, float* scales, unsigned* bad, hipStream_t s);
size_t packed_q8_bytes(int M, int K);
// greedy argmax per node; work: argmax_work_bytes(N, V) bytes of device scratch
size_t argmax_work_bytes(int N, int V);
hipError_t launch_argmax(const float* logits, int N, int V, int* g, void* work, hipStream_t s);
// per-row top-k (k <= kTopKMax, decreasing, lower index first on ties) and
// log-sum-exp (lse may be nullptr); work: topk_work_bytes(N, V) bytes
constexpr int kTopKMax = 8;
size_t topk_work_bytes(int N, int V);
hipError_t launch_topk(const float* logits, int N, int V, int k, int* idx, float* val, float* lse, void* work,
                       hipStream_t s);
// greedy accept from G per-workgroup (logit bits, token) maxima per node
// (parts [N][G][2], N <= 64): the argmax of every node, then the walk
hipError_t launch_greedy_from_parts(const unsigned* parts, int G, int N, const int* tokens, const int* parents,
                                    const int* depth, int* path, int* path_len, int* next, hipStream_t s);
hipError_t launch_greedy_walk(const int* tokens, const int* parents, const int* depth, int N, const int* g,
                              int* path, int* path_len, int* next, hipStream_t s);
// mode: 1 without replacement, 2 independent, 3 chosen, 4 CDF-first (3, 4: draft == nullptr);
// topk > 0 restricts the targets to each row's topk largest logits
// rejection sampling down the tree on ceil(V / 2048) workgroups that trade
// slice sums through work (sample_work_bytes(), zeroed once before the first
// use and then owned by the sampler: one call at a time per work area); on a
// wait that times out *path_len = 0 and err (if given) counts it
constexpr size_t kSampleWorkBytes = (64 + 64) * 4 + (size_t)2 * 64 * 4 * 8 + (size_t)2 * 64 * 256 * 4;
constexpr int kSampleMaxVocab = 64 * 2048;  // the sampling walk's vocabulary limit
size_t sample_work_bytes();
hipError_t launch_sample_accept(const int* tokens, const int* parents, int N, int V, const float* logits,
                                const float* draft, double temperature, uint64_t seed, int mode, int topk, void* work,
                                unsigned* err, int* path, int* path_len, int* next, hipStream_t s);
// inverse-CDF picks for CDF-first tree assembly: out[q] = the token drawn
// from softmax(logits[rows[q]] / T) (whole vocabulary V) at uniform U[q], by
// ascending token id
constexpr int kMaxPicks = 64;
struct CdfPickArgs {
  const float* logits;
  int V, n;
  float T;
  int rows[kMaxPicks];
  double U[kMaxPicks];
  int* out;
};
hipError_t launch_cdf_pick(const CdfPickArgs& a, hipStream_t s);
hipError_t launch_commit(int f32, void* kc, void* vc, const void* kt, const void* vt, int LH, int max_ctx,
                         int max_nodes, int DH, int P, const int* path, const int* path_len, unsigned* err,
                         hipStream_t s);

// ---- the persistent single-launch pass (fused.hip), bf16 models with head
// dimension 64 and at most kFMaxN nodes
constexpr int kFXcd = 8;                   // XCDs
constexpr int kFRanks = 32;                // compute workgroups per XCD
constexpr int kFGroups = kFXcd * kFRanks;  // compute workgroups (one per CU)
constexpr int kFMaxN = 64;                 // nodes
constexpr int kFAutoMaxN = 64;             // most nodes the default pass mode sends to it
constexpr int kFMaxL = 255;                // layers
// stages of a layer; their flags are [kFStages][kFGroups] words
enum FStage { FS_LN1 = 0, FS_QKV, FS_ATT, FS_WO, FS_LN2, FS_FC, FS_WPR, FS_SPARE, kFStages };
constexpr unsigned kFTagsPerPass = (unsigned)kFStages * (kFMaxL + 1);
constexpr int kFAttRows = 256;  // cache rows per attention unit (32 per wave of 8)
constexpr int kLwSlots = 12;  // per-layer parameter pointers (see LwSlot in fused.hip)
// plan row of one compute workgroup (int32): the rank's position in the
// order attention units are dealt in; per weight GEMM a count then row blocks;
// the LM-head row-block range
enum PlanSlot { PL_ATT = 0, PL_QKV = 9, PL_WO = 14, PL_FC = 19, PL_WPR = 24, PL_HEAD = 29, kPlanStride = 32 };
constexpr int kPlanMaxRb = 4;
// control words: pass counter, finished workgroups, abort flag, abort reason, claims [kFGroups]
enum { FZ_PASS = 0, FZ_DONE = 1, FZ_ABORT = 2, FZ_WHY = 3, FZ_CLAIM = 16, kFCtlWords = FZ_CLAIM + kFGroups };

struct FusedArgs {
  // model
  const void* const* lw;  // device [L][kLwSlots]: packed W_qkv, W_o, W_fc, W_pr, then biases, LN gains/biases
  const uint16_t *wte, *wpe, *lnf_g, *lnf_b;
  const void* p_head;     // packed tied LM head
  int L, d, H, M, V;
  float eps, scale;
  // session
  const uint16_t *kc, *vc;  // cache [L][H][max_ctx][64]
  uint16_t *kt, *vt;        // tree scratch [L][H][max_nodes][64]
  int max_ctx, max_nodes;
  const int* tree;          // staged tree (tokens, positions, depths, parents, offsets, path32, paths)
  int N, P;
  float* logits;            // [N][V]
  unsigned* head_part;      // [kFMaxN][kFGroups][2]: each workgroup's largest logit (bits) and its token per node
  // workspaces
  float* xr;                // [kFXcd][kFMaxN][d] residual stream, one copy per XCD
  float* q;                 // [kFMaxN][d]
  uint16_t *act1, *act2;    // [kFXcd][act_stride] LayerNorm outputs (float16 fragments), one copy per XCD
  size_t act_stride;
  uint16_t* fo;             // attention outputs, float16 fragments [4 tiles][d / 32][512]
  float* apart;             // attention parts [H][4 tiles][att_units + 1][16][68]: max, sum, -, -, output
  int att_units;            // prefix units of 256 cache rows: ceil(P / 256)
  unsigned* tile_ctr;       // [H][4 tiles]: attention units of the tile done in this layer (wraps to 0)
  uint16_t* ff;             // GELU outputs, float16 fragments [4 tiles][M / 32][512]
  long long* xacc;          // [3][kFMaxN][d] fixed-point (2^-32) sums of the residual GEMMs' partials
  unsigned* flags;          // [kFStages][kFGroups]
  unsigned* ctl;            // [kFCtlWords]
  const int* plan;          // [kFGroups][kPlanStride]
  int xh[2 * kFXcd];        // heads [xh[2x], xh[2x+1]) of XCD x
  int xf[2 * kFXcd];        // hidden k-steps [xf[2x], xf[2x+1]) of XCD x
  unsigned* err;            // session error counter
  unsigned long long timeout;  // s_memrealtime ticks (100 MHz) before a wait gives up
  unsigned long long* trace;  // stage timestamps [kFGroups][L + 1][kFStages][3], or nullptr
  int q8;                   // 8-bit weights: each packed matrix is 8-bit fragments followed by its row scales
  int l0;                   // the first layer the pass runs (0: from the embedding)
  const float* x_in;        // l0 > 0: [N][d] residual stream at layer l0's input (row = node slot)
};

// Work split of the fused pass for a model shape and 16-node tile count:
// tab receives [kFGroups][kPlanStride]; false (with a reason) if the shape
// does not fit the plan's limits.
bool fused_plan(int H, int d, int M, int V, int ntiles, int* tab, int* xh, int* xf, std::string* why);
size_t fused_lds_bytes(int L);
// raises the kernels' dynamic LDS limit (once per process, before the first launch)
hipError_t fused_prepare();
hipError_t launch_fused(const FusedArgs& a, hipStream_t s);

}  // namespace ssd
