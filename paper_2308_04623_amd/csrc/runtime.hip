// Host runtime of libssd: the C ABI declared in include/ssd.h.
//
// Validation and tree bookkeeping run on the host before anything is
// enqueued; the per-call tree description (tokens, positions, depths,
// parents, ancestor bitmask) is staged through pinned memory and copied to
// the device on the caller's stream; the pass is a fixed sequence of kernel
// launches on that stream, so it can be captured into a HIP graph.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/ssd.h"
#include "ssd_internal.h"

using namespace ssd;

namespace {

thread_local std::string g_last_error;


// Node counts up to this use the vector-ALU GEMM on the automatic path.
constexpr int kVecMaxNodes = 4;
constexpr int kMaxNodes = 1024;
constexpr int kStageSlots = 4;

ssd_status fail(ssd_status st, const std::string& msg) {
  g_last_error = msg;
  return st;
}

#define HIP_TRY(expr)                                                                          \
  do {                                                                                         \
    hipError_t e_ = (expr);                                                                    \
    if (e_ != hipSuccess)                                                                      \
      return fail(SSD_E_DEVICE, std::string(#expr) + ": " + hipGetErrorString(e_));            \
  } while (0)

int round_up(int a, int b) { return (a + b - 1) / b * b; }

}  // namespace

struct ssd_model {
  ssd_config cfg;
  int dh = 0;
  bool f32 = false;
  const void *wte = nullptr, *wpe = nullptr, *lnf_g = nullptr, *lnf_b = nullptr;
  std::vector<const void*> ln1_g, ln1_b, w_qkv, b_qkv, w_o, b_o, ln2_g, ln2_b, w_fc, b_fc, w_pr, b_pr;
  // bf16 only: packed copies
  void* pack = nullptr;
  bool owns_pack = true;  // false for a prefix view (shares its parent's copies)
  std::vector<const void*> p_qkv, p_o, p_fc, p_pr;
  const void* p_head = nullptr;
  // 8-bit models: the packed copies hold 8-bit fragments, with these per-row scales
  bool q8 = false;
  std::vector<const float*> s_qkv, s_o, s_fc, s_pr;
  const float* s_head = nullptr;
  void* wtab = nullptr;  // device [4][n_layer]: p_qkv, p_o, p_fc, p_pr (for the prefetcher); own copy per view
  void* ftab = nullptr;  // device [n_layer][kLwSlots]: the persistent pass's per-layer parameters; own copy per view
};

// the device table of a bf16 model's per-layer parameters for the persistent
// pass (see LwSlot in fused.hip)
static hipError_t make_ftab(ssd_model* m) {
  const int L = m->cfg.n_layer;
  std::vector<const void*> t;
  for (int l = 0; l < L; ++l) {
    const void* row[kLwSlots] = {m->p_qkv[l], m->p_o[l], m->p_fc[l], m->p_pr[l], m->b_qkv[l], m->b_o[l],
                                 m->b_fc[l],  m->b_pr[l], m->ln1_g[l], m->ln1_b[l], m->ln2_g[l], m->ln2_b[l]};
    t.insert(t.end(), row, row + kLwSlots);
  }
  hipError_t e = hipMalloc(&m->ftab, t.size() * sizeof(void*));
  if (e == hipSuccess) e = hipMemcpy(m->ftab, t.data(), t.size() * sizeof(void*), hipMemcpyHostToDevice);
  return e;
}

// the device table of a bf16 model's packed weight pointers, [4][L]
static hipError_t make_wtab(ssd_model* m) {
  const int L = m->cfg.n_layer;
  std::vector<const void*> t;
  for (auto* v : {&m->p_qkv, &m->p_o, &m->p_fc, &m->p_pr}) t.insert(t.end(), v->begin(), v->begin() + L);
  hipError_t e = hipMalloc(&m->wtab, t.size() * sizeof(void*));
  if (e == hipSuccess) e = hipMemcpy(m->wtab, t.data(), t.size() * sizeof(void*), hipMemcpyHostToDevice);
  return e;
}

struct ssd_kv {
  const ssd_model* m = nullptr;
  // per-session switches (ssd_kv_set_options)
  int gemm_path = 0;  // 0 auto, 1 vector ALU, 2 matrix cores
  int prefetch = 1;   // warm each weight GEMM's L2 from the kernel before it
  int pass_mode = 0;  // 0 auto, 1 one kernel per sub-layer, 2 the persistent single-launch pass only
  int max_ctx = 0, max_nodes = 0, npad = 0;
  void *kc = nullptr, *vc = nullptr, *kt = nullptr, *vt = nullptr;
  void* ws = nullptr;  // one device allocation for every workspace below
  float* x = nullptr;
  float* q = nullptr;
  void* act_a = nullptr;  // LN outputs [npad][d]
  void* act_o = nullptr;  // attention outputs [npad][d]
  void* act_f = nullptr;  // GELU outputs [npad][d_mlp]
  float* part = nullptr;  // split-K partial sums [kMaxSplits][max_nodes][d]
  float* apart = nullptr;  // attention partials (see AttnArgs::part)
  int* d_tree = nullptr;  // the staged tree (see stage_bytes)
  int* d_accept_tree = nullptr;  // tokens[N] parents[N] depth[N] for accept
  int* d_argmax = nullptr;
  void* d_amwork = nullptr;  // argmax / top-k partials
  void* d_sw = nullptr;   // the sampling walk's exchange area (sample_work_bytes, zeroed at creation)
  unsigned* d_err = nullptr;
  // pinned staging ring
  char* pinned = nullptr;
  size_t slot_bytes = 0;
  int next_slot = 0;
  hipEvent_t slot_ev[kStageSlots] = {};
  bool slot_used[kStageSlots] = {};
  // pass signals and the weight prefetcher (bf16 models)
  unsigned long long* d_sig = nullptr;  // bumped by every kernel of a pass as it starts
  unsigned* d_xcc0 = nullptr;           // XCD of block 0 of the last pass's embedding
  unsigned* d_sink = nullptr;
  unsigned long long sig_count = 0;     // signals of every pass enqueued so far
  hipStream_t pf_stream = nullptr;      // created on first use
  // the persistent single-launch pass (bf16 models, head dimension 64)
  bool fz_ok = false;                  // workspaces and plans exist
  void* fz_ws = nullptr;
  FusedArgs fz{};                      // workspace pointers, XCD ranges
  int* fz_plan[5] = {};                // device plans per 16-node tile count (1..4)
  // the last enqueued pass: where it left its residual stream (fz.xr or x),
  // its node count and its model's layer count (0: none yet)
  bool resid_fused = false;
  int last_n = 0, last_layers = 0;
};

struct ssd_graph {
  hipGraph_t graph = nullptr;
  hipGraphExec_t exec = nullptr;
  char* pinned = nullptr;
  const ssd_model* m = nullptr;  // the pass it replays
  ssd_kv* kv = nullptr;
  int n = 0;
  bool fused = false;   // captured as the persistent single launch
  int gemm_path = 0;    // the session's GEMM path at capture (fixes the prefetcher's plan)
};

// ------------------------------------------------------------------ small host helpers

extern "C" const char* ssd_status_string(ssd_status s) {
  switch (s) {
    case SSD_OK: return "ok";
    case SSD_E_INVALID_ARG: return "invalid argument";
    case SSD_E_INVALID_TREE: return "invalid tree";
    case SSD_E_CAPACITY: return "capacity exceeded";
    case SSD_E_DEVICE: return "device error";
    case SSD_E_UNSUPPORTED: return "unsupported shape";
  }
  return "unknown status";
}

extern "C" const char* ssd_last_error(void) { return g_last_error.c_str(); }

extern "C" ssd_status ssd_kv_set_options(ssd_kv* kv, const ssd_options* opt) {
  if (!kv || !opt) return fail(SSD_E_INVALID_ARG, "null argument");
  if (opt->pass_mode < 0 || opt->pass_mode > 2) return fail(SSD_E_INVALID_ARG, "pass mode must be 0, 1 or 2");
  if (opt->gemm_path < 0 || opt->gemm_path > 2) return fail(SSD_E_INVALID_ARG, "gemm path must be 0, 1 or 2");
  if (opt->weight_prefetch != 0 && opt->weight_prefetch != 1)
    return fail(SSD_E_INVALID_ARG, "weight prefetch must be 0 or 1");
  kv->pass_mode = opt->pass_mode;
  kv->gemm_path = opt->gemm_path;
  kv->prefetch = opt->weight_prefetch;
  return SSD_OK;
}

extern "C" ssd_status ssd_kv_get_options(const ssd_kv* kv, ssd_options* opt) {
  if (!kv || !opt) return fail(SSD_E_INVALID_ARG, "null argument");
  opt->pass_mode = kv->pass_mode;
  opt->gemm_path = kv->gemm_path;
  opt->weight_prefetch = kv->prefetch;
  return SSD_OK;
}

extern "C" ssd_status ssd_kv_set_trace(ssd_kv* kv, uint64_t* buf) {
  if (!kv) return fail(SSD_E_INVALID_ARG, "null session");
  if (!kv->fz_ok) return fail(SSD_E_UNSUPPORTED, "the session has no persistent pass");
  kv->fz.trace = (unsigned long long*)buf;
  return SSD_OK;
}

extern "C" ssd_status ssd_fused_plan(int32_t n_head, int32_t d_model, int32_t d_mlp, int32_t vocab, int32_t n_tiles,
                                      int32_t* tab, int32_t* xh, int32_t* xf) {
  if (!tab || !xh || !xf) return fail(SSD_E_INVALID_ARG, "null output");
  if (n_head <= 0 || d_model <= 0 || d_mlp <= 0 || vocab <= 0) return fail(SSD_E_INVALID_ARG, "sizes must be positive");
  std::string why;
  if (!fused_plan(n_head, d_model, d_mlp, vocab, n_tiles, tab, xh, xf, &why)) return fail(SSD_E_UNSUPPORTED, why);
  return SSD_OK;
}

extern "C" ssd_status ssd_validate_tree(const int32_t* tokens, const int32_t* parent_idx, int32_t n, int32_t vocab,
                                        int32_t* max_depth) {
  if (!tokens || !parent_idx) return fail(SSD_E_INVALID_ARG, "null tree array");
  if (n <= 0) return fail(SSD_E_INVALID_ARG, "n_nodes must be positive");
  if (parent_idx[0] != -1) return fail(SSD_E_INVALID_TREE, "parent_idx[0] must be -1");
  std::vector<int32_t> depth(n, 0);
  int32_t md = 0;
  for (int32_t i = 0; i < n; ++i) {
    if (tokens[i] < 0 || tokens[i] >= vocab)
      return fail(SSD_E_INVALID_ARG, "token " + std::to_string(i) + " out of range");
    if (i > 0) {
      const int32_t p = parent_idx[i];
      if (p < 0 || p >= i) return fail(SSD_E_INVALID_TREE, "parent_idx[" + std::to_string(i) + "] not in [0, i)");
      depth[i] = depth[p] + 1;
      md = std::max(md, depth[i]);
    }
  }
  if (max_depth) *max_depth = md;
  return SSD_OK;
}

extern "C" ssd_status ssd_tree_prep(const int32_t* parent_idx, int32_t n, int32_t* depth, uint64_t* anc) {
  if (!parent_idx || n <= 0) return fail(SSD_E_INVALID_ARG, "bad tree arguments");
  if (parent_idx[0] != -1) return fail(SSD_E_INVALID_TREE, "parent_idx[0] must be -1");
  for (int32_t i = 1; i < n; ++i)
    if (parent_idx[i] < 0 || parent_idx[i] >= i) return fail(SSD_E_INVALID_TREE, "parent_idx not in [0, i)");
  const int W = (n + 63) / 64;
  std::vector<int32_t> dep(n, 0);
  for (int32_t i = 0; i < n; ++i) {
    uint64_t* row = anc ? anc + (size_t)i * W : nullptr;
    if (i == 0) {
      if (row) std::fill(row, row + W, 0ull);
    } else {
      const int32_t p = parent_idx[i];
      dep[i] = dep[p] + 1;
      if (row) std::copy(anc + (size_t)p * W, anc + (size_t)p * W + W, row);  // ancestors of the parent
    }
    if (row) row[i >> 6] |= 1ull << (i & 63);
  }
  if (depth) std::copy(dep.begin(), dep.end(), depth);
  return SSD_OK;
}

// ------------------------------------------------------------------ model

static bool cfg_ok(const ssd_config* c, std::string* why) {
  if (!c) return *why = "null config", false;
  if (c->n_layer <= 0 || c->d_model <= 0 || c->n_head <= 0 || c->d_mlp <= 0 || c->vocab <= 0 || c->n_pos <= 0)
    return *why = "config sizes must be positive", false;
  if (c->d_model % c->n_head) return *why = "d_model must divide by n_head", false;
  if (c->dtype != SSD_F32 && c->dtype != SSD_BF16) return *why = "dtype must be SSD_F32 or SSD_BF16", false;
  return true;
}

static ssd_status model_create(const ssd_config* cfg, const ssd_weights* w, void* stream, ssd_model** out, bool q8) {
  std::string why;
  if (!out || !w) return fail(SSD_E_INVALID_ARG, "null argument");
  if (!cfg_ok(cfg, &why)) return fail(SSD_E_INVALID_ARG, why);
  const int d = cfg->d_model, dh = d / cfg->n_head, L = cfg->n_layer;
  if (d % 32 || cfg->d_mlp % 32 || (dh != 32 && dh != 64))
    return fail(SSD_E_UNSUPPORTED, "need d_model % 32 == 0, d_mlp % 32 == 0, head_dim 32 or 64");
  if (q8 && cfg->dtype != SSD_BF16) return fail(SSD_E_UNSUPPORTED, "8-bit weights are made from a bfloat16 model");
  if (q8 && (d % 64 || cfg->d_mlp % 64)) return fail(SSD_E_UNSUPPORTED, "8-bit weights need d_model, d_mlp % 64 == 0");
  if (!w->wte || !w->wpe || !w->lnf_g || !w->lnf_b) return fail(SSD_E_INVALID_ARG, "null embedding / ln_f pointer");
  const void* const* per[12] = {w->ln1_g, w->ln1_b, w->w_qkv, w->b_qkv, w->w_o, w->b_o,
                                w->ln2_g, w->ln2_b, w->w_fc, w->b_fc, w->w_pr, w->b_pr};
  for (auto a : per) {
    if (!a) return fail(SSD_E_INVALID_ARG, "null per-layer pointer array");
    for (int l = 0; l < L; ++l)
      if (!a[l]) return fail(SSD_E_INVALID_ARG, "null per-layer parameter pointer");
  }
  ssd_model* m = new ssd_model();
  m->cfg = *cfg;
  m->dh = dh;
  m->f32 = cfg->dtype == SSD_F32;
  m->wte = w->wte;
  m->wpe = w->wpe;
  m->lnf_g = w->lnf_g;
  m->lnf_b = w->lnf_b;
  std::vector<const void*>* dst[12] = {&m->ln1_g, &m->ln1_b, &m->w_qkv, &m->b_qkv, &m->w_o, &m->b_o,
                                       &m->ln2_g, &m->ln2_b, &m->w_fc, &m->b_fc, &m->w_pr, &m->b_pr};
  for (int i = 0; i < 12; ++i) dst[i]->assign(per[i], per[i] + L);
  if (!m->f32) {
    const int M = cfg->d_mlp, V = cfg->vocab;
    m->q8 = q8;
    auto pbytes = [&](int rows, int K) { return q8 ? packed_q8_bytes(rows, K) : packed_bytes(rows, K); };
    // per-row scales of the 8-bit copies: [ceil(rows/16) 16] float32, 256-byte aligned
    auto sbytes = [&](int rows) { return q8 ? (size_t)round_up(round_up(rows, 16) * 4, 256) : (size_t)0; };
    const size_t b_qkv = pbytes(3 * d, d), b_o = pbytes(d, d), b_fc = pbytes(M, d), b_pr = pbytes(d, M),
                 b_head = pbytes(V, d);
    const size_t total = (b_qkv + b_o + b_fc + b_pr + sbytes(3 * d) + 2 * sbytes(d) + sbytes(M)) * L + b_head +
                         sbytes(V);
    // the packed copies (and scales), then one counter of weights past
    // float16's range (8-bit copies: of rows holding a NaN or infinity)
    hipError_t e = hipMalloc(&m->pack, total + 256);
    if (e != hipSuccess) {
      delete m;
      return fail(SSD_E_DEVICE, std::string("hipMalloc(packed weights): ") + hipGetErrorString(e));
    }
    hipStream_t s = (hipStream_t)stream;
    unsigned* bad = (unsigned*)((char*)m->pack + total);
    e = hipMemsetAsync(bad, 0, 4, s);
    char* p = (char*)m->pack;
    // (8-bit: the fragments first, then the row scales)
    auto pack = [&](const void* src, int rows, int cols, size_t bytes, std::vector<const float*>* sc) -> const void* {
      const void* r = p;
      if (!q8) {
        if (e == hipSuccess) e = launch_pack_bf16((const uint16_t*)src, rows, cols, p, bad, s);
        p += bytes;
        return r;
      }
      float* scales = (float*)(p + bytes);
      if (e == hipSuccess) e = launch_pack_q8((const uint16_t*)src, rows, cols, p, scales, bad, s);
      sc->push_back(scales);
      p += bytes + sbytes(rows);
      return r;
    };
    std::vector<const float*> s_head;
    for (int l = 0; l < L; ++l) {
      m->p_qkv.push_back(pack(m->w_qkv[l], 3 * d, d, b_qkv, &m->s_qkv));
      m->p_o.push_back(pack(m->w_o[l], d, d, b_o, &m->s_o));
      m->p_fc.push_back(pack(m->w_fc[l], M, d, b_fc, &m->s_fc));
      m->p_pr.push_back(pack(m->w_pr[l], d, M, b_pr, &m->s_pr));
    }
    m->p_head = pack(m->wte, V, d, b_head, &s_head);
    if (q8) m->s_head = s_head[0];
    unsigned n_bad = 0;
    if (e == hipSuccess) e = hipMemcpyAsync(&n_bad, bad, 4, hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e == hipSuccess && n_bad) {
      (void)hipFree(m->pack);
      delete m;
      return fail(SSD_E_UNSUPPORTED, q8 ? "a weight is NaN or infinite: it has no 8-bit code"
                                        : "a weight's magnitude exceeds 65504 (or is NaN): the matrix cores take "
                                          "float16 copies of the weights");
    }
    if (e == hipSuccess) e = make_wtab(m);
    if (e == hipSuccess) e = make_ftab(m);
    if (e != hipSuccess) {
      (void)hipFree(m->pack);
      if (m->wtab) (void)hipFree(m->wtab);
      if (m->ftab) (void)hipFree(m->ftab);
      delete m;
      return fail(SSD_E_DEVICE, std::string("weight packing: ") + hipGetErrorString(e));
    }
  }
  *out = m;
  return SSD_OK;
}

extern "C" ssd_status ssd_model_create(const ssd_config* cfg, const ssd_weights* w, void* stream, ssd_model** out) {
  return model_create(cfg, w, stream, out, false);
}

extern "C" ssd_status ssd_model_create_q8(const ssd_config* cfg, const ssd_weights* w, void* stream,
                                          ssd_model** out) {
  return model_create(cfg, w, stream, out, true);
}

extern "C" void ssd_model_destroy(ssd_model* m) {
  if (!m) return;
  if (m->pack && m->owns_pack) (void)hipFree(m->pack);
  if (m->wtab) (void)hipFree(m->wtab);
  if (m->ftab) (void)hipFree(m->ftab);
  delete m;
}

extern "C" ssd_status ssd_model_prefix_view(const ssd_model* m, int32_t n_layer, ssd_model** out) {
  if (!m || !out) return fail(SSD_E_INVALID_ARG, "null argument");
  if (n_layer < 1 || n_layer > m->cfg.n_layer) return fail(SSD_E_INVALID_ARG, "n_layer outside [1, model layers]");
  ssd_model* v = new ssd_model(*m);
  v->cfg.n_layer = n_layer;
  v->owns_pack = false;
  std::vector<const void*>* per[] = {&v->ln1_g, &v->ln1_b, &v->w_qkv, &v->b_qkv, &v->w_o, &v->b_o, &v->ln2_g,
                                     &v->ln2_b, &v->w_fc, &v->b_fc, &v->w_pr, &v->b_pr};
  for (auto a : per) a->resize(n_layer);
  v->wtab = nullptr;
  v->ftab = nullptr;
  if (!v->f32) {
    v->p_qkv.resize(n_layer);
    v->p_o.resize(n_layer);
    v->p_fc.resize(n_layer);
    v->p_pr.resize(n_layer);
    if (v->q8) {
      v->s_qkv.resize(n_layer);
      v->s_o.resize(n_layer);
      v->s_fc.resize(n_layer);
      v->s_pr.resize(n_layer);
    }
    hipError_t e = make_wtab(v);
    if (e == hipSuccess) e = make_ftab(v);
    if (e != hipSuccess) {
      if (v->wtab) (void)hipFree(v->wtab);
      if (v->ftab) (void)hipFree(v->ftab);
      delete v;
      return fail(SSD_E_DEVICE, std::string("weight table: ") + hipGetErrorString(e));
    }
  }
  *out = v;
  return SSD_OK;
}

// ------------------------------------------------------------------ session

extern "C" ssd_status ssd_kv_bytes(const ssd_config* cfg, int32_t max_ctx, int32_t max_nodes, size_t* cache_bytes,
                                   size_t* tree_bytes) {
  std::string why;
  if (!cfg_ok(cfg, &why)) return fail(SSD_E_INVALID_ARG, why);
  if (max_ctx < 0 || max_nodes <= 0) return fail(SSD_E_INVALID_ARG, "bad sizes");
  const size_t es = cfg->dtype == SSD_F32 ? 4 : 2;
  const size_t per_row = (size_t)cfg->n_layer * cfg->d_model * es;  // all heads of all layers
  if (cache_bytes) *cache_bytes = per_row * max_ctx;
  if (tree_bytes) *tree_bytes = per_row * max_nodes;
  return SSD_OK;
}

// staged tree: tokens, positions, depths, parents, root-path offsets
// (max_nodes each), then the root paths themselves (at most n(n+1)/2 entries)
// Staged tree: tokens, positions, depths, parents, root-path offsets
// ([max_nodes] each); then for the n nodes the first kPath32 entries of each
// root path ([n][kPath32], root first, padded with the node itself); then all
// root paths back to back (offsets above).
static size_t stage_bytes(int max_nodes) {
  return (size_t)5 * max_nodes * 4 + (size_t)max_nodes * kPath32 * 4 + (size_t)max_nodes * (max_nodes + 1) / 2 * 4;
}

// Workspaces and work plans of the persistent pass.  The pass needs one
// workgroup per CU on 8 XCDs of 32 CUs and head dimension 64; otherwise the
// session keeps only the per-sub-layer kernels (fz_ok stays false).
static ssd_status fused_setup(ssd_kv* kv) {
  const ssd_model* m = kv->m;
  const ssd_config& c = m->cfg;
  if (m->dh != 64 || c.d_model > 2048 || c.n_layer > kFMaxL) return SSD_OK;
  int dev = 0, cus = 0;
  HIP_TRY(hipGetDevice(&dev));
  HIP_TRY(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev));
  if (cus != kFGroups) return SSD_OK;
  const int d = c.d_model, M = c.d_mlp;
  std::vector<int> tabs((size_t)4 * kFGroups * kPlanStride);
  FusedArgs& a = kv->fz;
  std::string why;
  for (int nt = 1; nt <= 4; ++nt)
    if (!fused_plan(c.n_head, d, M, c.vocab, nt, tabs.data() + (size_t)(nt - 1) * kFGroups * kPlanStride, a.xh,
                    a.xf, &why))
      return SSD_OK;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    size_t o = off;
    off += (bytes + 255) / 256 * 256;
    return o;
  };
  const size_t act_stride = (size_t)kFMaxN * d;  // float16 elements of one XCD's copy
  const size_t o_xr = take((size_t)kFXcd * kFMaxN * d * 4), o_q = take((size_t)kFMaxN * d * 4);
  const size_t o_a1 = take(kFXcd * act_stride * 2), o_a2 = take(kFXcd * act_stride * 2);
  const size_t o_fo = take((size_t)kFMaxN * d * 2), o_ff = take((size_t)kFMaxN * M * 2);
  const size_t att_parts = (size_t)(kv->max_ctx + kFAttRows - 1) / kFAttRows + 1;
  const size_t o_ap = take((size_t)c.n_head * 4 * att_parts * 16 * 68 * 4);
  const size_t o_xs = take((size_t)3 * kFMaxN * d * 8);
  const size_t o_fl = take((size_t)kFStages * kFGroups * 4), o_ctl = take((size_t)kFCtlWords * 4);
  const size_t o_plan = take(tabs.size() * 4);
  const size_t o_tc = take((size_t)c.n_head * 4 * 4);
  const size_t o_hp = take((size_t)kFMaxN * kFGroups * 8);
  static const hipError_t prep = fused_prepare();
  if (prep != hipSuccess) return SSD_OK;  // keep the per-sub-layer kernels
  HIP_TRY(hipMalloc(&kv->fz_ws, off));
  HIP_TRY(hipMemset(kv->fz_ws, 0, off));
  HIP_TRY(hipMemcpy((char*)kv->fz_ws + o_plan, tabs.data(), tabs.size() * 4, hipMemcpyHostToDevice));
  char* b = (char*)kv->fz_ws;
  a.xr = (float*)(b + o_xr);
  a.q = (float*)(b + o_q);
  a.act1 = (uint16_t*)(b + o_a1);
  a.act2 = (uint16_t*)(b + o_a2);
  a.act_stride = act_stride;
  a.fo = (uint16_t*)(b + o_fo);
  a.ff = (uint16_t*)(b + o_ff);
  a.apart = (float*)(b + o_ap);
  a.xacc = (long long*)(b + o_xs);
  a.flags = (unsigned*)(b + o_fl);
  a.ctl = (unsigned*)(b + o_ctl);
  a.tile_ctr = (unsigned*)(b + o_tc);
  a.head_part = (unsigned*)(b + o_hp);
  for (int nt = 1; nt <= 4; ++nt) kv->fz_plan[nt] = (int*)(b + o_plan) + (size_t)(nt - 1) * kFGroups * kPlanStride;
  a.err = kv->d_err;
  a.timeout = 20000000ull;  // 200 ms
  kv->fz_ok = true;
  return SSD_OK;
}

// whether a verification pass of model m over n nodes runs as the persistent single launch
static bool use_fused(const ssd_model* m, const ssd_kv* kv, int n) {
  if (kv->pass_mode == 1 || m->f32 || !kv->fz_ok || !m->ftab) return false;
  // the persistent pass is forced, or chosen where it is the faster one
  // (measured on the GPT-2-L shape: at every node count it supports)
  return kv->pass_mode == 2 ? n <= kFMaxN : n <= kFAutoMaxN;
}

extern "C" ssd_status ssd_verify_path(const ssd_model* m, const ssd_kv* kv, int32_t n, int32_t* path) {
  if (!m || !kv || !path || n < 1 || n > kv->max_nodes) return fail(SSD_E_INVALID_ARG, "bad argument");
  *path = use_fused(m, kv, n) ? 2 : 1;
  return SSD_OK;
}

extern "C" ssd_status ssd_kv_create(const ssd_model* m, int32_t max_ctx, int32_t max_nodes, void* k_cache,
                                    void* v_cache, void* k_tree, void* v_tree, ssd_kv** out) {
  if (!m || !out || !k_tree || !v_tree) return fail(SSD_E_INVALID_ARG, "null argument");
  if (max_ctx < 0 || max_nodes <= 0) return fail(SSD_E_INVALID_ARG, "bad sizes");
  if (max_ctx > 0 && (!k_cache || !v_cache)) return fail(SSD_E_INVALID_ARG, "null cache with max_ctx > 0");
  if (max_nodes > kMaxNodes) return fail(SSD_E_CAPACITY, "max_nodes above 1024");
  const ssd_config& c = m->cfg;
  ssd_kv* kv = new ssd_kv();
  kv->m = m;
  kv->max_ctx = max_ctx;
  kv->max_nodes = max_nodes;
  kv->kc = k_cache;
  kv->vc = v_cache;
  kv->kt = k_tree;
  kv->vt = v_tree;
  // GEMMs read activation rows in power-of-two node tiles (16..256), or in
  // groups of 256 beyond that, so pad the row count to cover the last tile.
  if (max_nodes <= 256) {
    int p2 = 16;
    while (p2 < max_nodes) p2 *= 2;
    kv->npad = p2;
  } else {
    kv->npad = round_up(max_nodes, 256);
  }
  const size_t es = m->f32 ? 4 : 2;
  const int d = c.d_model, M = c.d_mlp, V = c.vocab;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    size_t o = off;
    off += (bytes + 255) / 256 * 256;
    return o;
  };
  const size_t o_x = take((size_t)max_nodes * d * 4), o_q = take((size_t)max_nodes * d * 4);
  // GEMM inputs: fp32 rows (fp32 models) or float16 fragments (bf16 models)
  const size_t planes = 1;
  const size_t o_a = take(planes * kv->npad * d * es), o_o = take(planes * kv->npad * d * es);
  const size_t o_f = take(planes * kv->npad * M * es);
  const size_t o_part = take((size_t)kMaxSplits * max_nodes * d * 4);  // split-K partials
  // attention partials: fp32 models (H, 64-row tiles, node, DH + 2); bf16
  // models (H, prefix chunks, node, DH + 4)
  const size_t ap_f32 = (size_t)c.n_head * ((max_ctx + 63) / 64) * max_nodes * (m->dh + 2);
  const size_t ap_bf16 = (size_t)c.n_head * attn_max_nsplit(max_ctx, c.n_head) * max_nodes * (m->dh + 4);
  const size_t o_apart = take((m->f32 ? ap_f32 : ap_bf16) * 4);
  const size_t o_tree = take(stage_bytes(max_nodes));
  const size_t o_at = take((size_t)3 * max_nodes * 4), o_am = take((size_t)max_nodes * 4);
  const size_t o_amw = take(std::max(argmax_work_bytes(max_nodes, V), topk_work_bytes(max_nodes, V)));
  const size_t o_sw = take(sample_work_bytes());
  const size_t o_err = take(256);
  const size_t o_sig = take(256);  // signal counter, XCD of block 0, sink
  hipError_t e = hipMalloc(&kv->ws, off);
  if (e == hipSuccess) e = hipMemset(kv->ws, 0, off);
  if (e != hipSuccess) {
    if (kv->ws) (void)hipFree(kv->ws);
    delete kv;
    return fail(SSD_E_DEVICE, std::string("workspace allocation: ") + hipGetErrorString(e));
  }
  char* b = (char*)kv->ws;
  kv->x = (float*)(b + o_x);
  kv->q = (float*)(b + o_q);
  kv->act_a = b + o_a;
  kv->act_o = b + o_o;
  kv->act_f = b + o_f;
  kv->part = (float*)(b + o_part);
  kv->apart = (float*)(b + o_apart);
  kv->d_tree = (int*)(b + o_tree);
  kv->d_accept_tree = (int*)(b + o_at);
  kv->d_argmax = (int*)(b + o_am);
  kv->d_amwork = b + o_amw;
  kv->d_sw = b + o_sw;
  kv->d_err = (unsigned*)(b + o_err);
  kv->d_sig = (unsigned long long*)(b + o_sig);
  kv->d_xcc0 = (unsigned*)(b + o_sig + 8);
  kv->d_sink = (unsigned*)(b + o_sig + 16);
  kv->slot_bytes = (stage_bytes(max_nodes) + 255) / 256 * 256;
  e = hipHostMalloc((void**)&kv->pinned, kv->slot_bytes * kStageSlots, hipHostMallocDefault);
  for (int i = 0; i < kStageSlots && e == hipSuccess; ++i) e = hipEventCreateWithFlags(&kv->slot_ev[i], hipEventDisableTiming);
  if (e != hipSuccess) {
    ssd_kv_destroy(kv);
    return fail(SSD_E_DEVICE, std::string("staging allocation: ") + hipGetErrorString(e));
  }
  if (!m->f32) {
    const ssd_status fs = fused_setup(kv);
    if (fs != SSD_OK) {
      ssd_kv_destroy(kv);
      return fs;
    }
  }
  *out = kv;
  return SSD_OK;
}

extern "C" void ssd_kv_destroy(ssd_kv* kv) {
  if (!kv) return;
  if (kv->pf_stream) {
    (void)hipStreamSynchronize(kv->pf_stream);
    (void)hipStreamDestroy(kv->pf_stream);
  }
  for (int i = 0; i < kStageSlots; ++i)
    if (kv->slot_ev[i]) {
      (void)hipEventSynchronize(kv->slot_ev[i]);
      (void)hipEventDestroy(kv->slot_ev[i]);
    }
  if (kv->pinned) (void)hipHostFree(kv->pinned);
  if (kv->ws) (void)hipFree(kv->ws);
  if (kv->fz_ws) (void)hipFree(kv->fz_ws);
  delete kv;
}

// Picks a pinned staging slot that no pending copy still reads.  Inside a
// stream capture the caller supplies its own buffer instead.
static ssd_status acquire_slot(ssd_kv* kv, char** host, int* slot) {
  const int i = kv->next_slot;
  kv->next_slot = (kv->next_slot + 1) % kStageSlots;
  if (kv->slot_used[i]) HIP_TRY(hipEventSynchronize(kv->slot_ev[i]));
  *host = kv->pinned + (size_t)i * kv->slot_bytes;
  *slot = i;
  return SSD_OK;
}

static ssd_status release_slot(ssd_kv* kv, int slot, hipStream_t s) {
  if (slot < 0) return SSD_OK;
  HIP_TRY(hipEventRecord(kv->slot_ev[slot], s));
  kv->slot_used[slot] = true;
  return SSD_OK;
}

// ------------------------------------------------------------------ verification pass

// A session's workspaces and cache are sized for its model; another model may
// use it only if every shape equals the session model's, except that it may
// have fewer layers (a draft view).
static bool same_shape_prefix(const ssd_config& a, const ssd_config& b) {
  return a.d_model == b.d_model && a.n_head == b.n_head && a.d_mlp == b.d_mlp && a.vocab == b.vocab &&
         a.dtype == b.dtype && a.n_layer <= b.n_layer;
}

static ssd_status check_verify_args(const ssd_model* m, const ssd_kv* kv, int32_t P, const int32_t* tokens,
                                    const int32_t* parents, int32_t n, const float* logits, int32_t* max_depth) {
  if (!m || !kv || !tokens || !parents || !logits) return fail(SSD_E_INVALID_ARG, "null argument");
  if (kv->m != m && !same_shape_prefix(m->cfg, kv->m->cfg))
    return fail(SSD_E_INVALID_ARG, "the model's shape differs from the session's (only a layer prefix may be used)");
  if (n <= 0) return fail(SSD_E_INVALID_ARG, "n_nodes must be positive");
  if (P < 0) return fail(SSD_E_INVALID_ARG, "negative prefix_len");
  if (n > kv->max_nodes) return fail(SSD_E_CAPACITY, "n_nodes above the session's max_nodes");
  if (P > kv->max_ctx) return fail(SSD_E_CAPACITY, "prefix_len above the session's max_ctx");
  ssd_status st = ssd_validate_tree(tokens, parents, n, m->cfg.vocab, max_depth);
  if (st != SSD_OK) return st;
  if (P + *max_depth >= m->cfg.n_pos) return fail(SSD_E_CAPACITY, "prefix_len + tree depth past the position table");
  return SSD_OK;
}

// Fills a staging buffer (see stage_bytes); returns the bytes used.
static size_t fill_stage(char* host, int P, const int32_t* tokens, const int32_t* parents, int n, int max_nodes) {
  int32_t* t = (int32_t*)host;
  int32_t* pos = t + max_nodes;
  int32_t* dep = pos + max_nodes;
  int32_t* par = dep + max_nodes;
  int32_t* off = par + max_nodes;
  int32_t* p32 = off + max_nodes;
  int32_t* paths = p32 + (size_t)n * kPath32;
  ssd_tree_prep(parents, n, dep, nullptr);  // validated by the caller
  int32_t total = 0;
  for (int i = 0; i < n; ++i) {
    t[i] = tokens[i];
    pos[i] = P + dep[i];
    par[i] = parents[i];
    off[i] = total;
    // root path of node i: walk up, filling from the end
    int32_t j = i;
    for (int k = dep[i]; k >= 0; --k) {
      paths[total + k] = j;
      j = parents[j];
    }
    for (int k = 0; k < kPath32; ++k) p32[(size_t)i * kPath32 + k] = paths[total + std::min(k, (int)dep[i])];
    total += dep[i] + 1;
  }
  return (size_t)5 * max_nodes * 4 + (size_t)n * kPath32 * 4 + (size_t)total * 4;
}

// One weight GEMM of the pass over n nodes: fp32 models use the plain
// kernel; bf16 models the vector-ALU kernel for few nodes (or when pinned)
// and the matrix-core kernel otherwise, in node groups of 16 / 256.
static int gemm_vec(int path, int n) { return (path == 0 ? (n <= kVecMaxNodes ? 1 : 2) : path) == 1; }

// k-steps per split of a weight GEMM over n nodes (one k-split for every
// node group, so all nodes leave the same partials)
static int gemm_kcs(int path, int n, int kind, int rows, int K) {
  const int vec = gemm_vec(path, n);
  int S = 1;
  return gemm_split_kc(rows, K, std::min(n, vec ? 16 : 256), vec, kind == EPI_PARTIAL, &S);
}

// The prefetcher's plan for a bf16 pass over n nodes: the launch geometry of
// the first launch of each weight GEMM (see run_gemm), the weight table and
// the session's signal words; base is filled in when the pass is enqueued.
static PrefetchPlan prefetch_plan(const ssd_model* m, const ssd_kv* kv, int path, int n) {
  PrefetchPlan pp{};
  const int d = m->cfg.d_model, M = m->cfg.d_mlp;
  const int vec = gemm_vec(path, n), nn = std::min(n, vec ? 16 : 256);
  const int kinds[4] = {EPI_QKV, EPI_PARTIAL, EPI_GELU, EPI_PARTIAL};
  const int rows[4] = {3 * d, d, M, d}, Ks[4] = {d, d, d, M};
  for (int k = 0; k < 4; ++k) {
    const GemmGeom g = gemm_geom(kinds[k], vec, rows[k], Ks[k], nn, gemm_kcs(path, n, kinds[k], rows[k], Ks[k]));
    // (the prefetcher reads 1 KB fragments: an 8-bit row block is KC / 2 of
    // them, K being a multiple of 64; a split's range rounds to whole ones)
    if (m->q8) pp.geo[k] = PfGeom{g.KC / 2, g.RBtot, g.RB, (g.kcs + 1) / 2, g.gx, g.gx * g.gy};
    else pp.geo[k] = PfGeom{g.KC, g.RBtot, g.RB, g.kcs, g.gx, g.gx * g.gy};
  }
  pp.W = (const void* const*)m->wtab;
  pp.L = m->cfg.n_layer;
  pp.sig = kv->d_sig;
  pp.xcc0 = kv->d_xcc0;
  pp.timeout = 5000000ull;  // 50 ms
  pp.sink = kv->d_sink;
  pp.magic = 0x5bd1e995u;
  return pp;
}

// Accounts for the signals of one bf16 pass about to be enqueued and, when
// weight prefetch is on, launches its prefetcher on the session's side
// stream first (the pass never waits for it).
static bool use_fused(const ssd_model* m, const ssd_kv* kv, int n);

static ssd_status start_pass_prefetch(const ssd_model* m, ssd_kv* kv, int n, bool fused, int path) {
  if (m->f32 || fused) return SSD_OK;
  const unsigned long long base = kv->sig_count;
  kv->sig_count += (unsigned long long)sigs_per_pass(m->cfg.n_layer);
  if (!kv->prefetch) return SSD_OK;
  if (!kv->pf_stream) HIP_TRY(hipStreamCreateWithFlags(&kv->pf_stream, hipStreamNonBlocking));
  PrefetchPlan pp = prefetch_plan(m, kv, path, n);
  pp.base = base;
  HIP_TRY(launch_prefetcher(pp, kv->pf_stream));
  return SSD_OK;
}

static hipError_t run_gemm(const ssd_model* m, int path, int n, int kind, const void* Wraw, const void* Wp,
                           const float* wscale, int rows, int K, const void* act, const Epi& ep, hipStream_t s) {
  if (m->f32) return launch_gemm_f32(kind, (const float*)Wraw, rows, K, (const float*)act, K, ep, s);
  const int vec = gemm_vec(path, n);
  const int group = vec ? 16 : 256;
  const int kcs = gemm_kcs(path, n, kind, rows, K);
  for (int n0 = 0; n0 < n; n0 += group) {
    Epi e2 = ep;
    e2.node0 = n0;
    e2.N = std::min(group, n - n0);
    // fragment tiles of 16 nodes, each K/32 fragments of 512 elements
    const uint16_t* a = (const uint16_t*)act + (size_t)(n0 / 16) * (K / 32) * 512;
    e2.sig = n0 == 0 ? ep.sig : nullptr;  // one signal per GEMM
    e2.wscale = m->q8 ? wscale : nullptr;
    hipError_t r = launch_gemm_bf16(kind, vec, Wp, rows, K, a, kcs, e2, s);
    if (r != hipSuccess) return r;
  }
  return hipSuccess;
}

// number of split-K partials a residual GEMM leaves for the next LayerNorm
static int resid_splits(const ssd_model* m, int path, int n, int rows, int K) {
  if (m->f32) return 0;
  const int vec = gemm_vec(path, n);
  int S = 1;
  gemm_split_kc(rows, K, std::min(n, vec ? 16 : 256), vec, 1, &S);
  return S;
}

// l0 > 0: the pass starts at layer l0 from the residual stream x_in
// ([n][d] fp32, device), the tree scratch already holding the nodes' K/V of
// layers below l0.
static ssd_status enqueue_verify(const ssd_model* m, ssd_kv* kv, int32_t P, int32_t n, const char* stage_host,
                                 size_t stage_used, float* logits, hipStream_t s, int l0 = 0,
                                 const float* x_in = nullptr) {
  const ssd_config& c = m->cfg;
  const int d = c.d_model, H = c.n_head, DH = m->dh, M = c.d_mlp, V = c.vocab, L = c.n_layer;
  const int maxn = kv->max_nodes;
  const int f32 = m->f32 ? 1 : 0;
  const size_t es = f32 ? 4 : 2;
  HIP_TRY(hipMemcpyAsync(kv->d_tree, stage_host, stage_used, hipMemcpyHostToDevice, s));
  const int* d_tok = kv->d_tree;
  const int* d_pos = kv->d_tree + maxn;
  const int* d_dep = kv->d_tree + 2 * maxn;
  const int* d_off = kv->d_tree + 4 * maxn;
  const int* d_path32 = kv->d_tree + 5 * maxn;
  const int* d_paths = d_path32 + (size_t)n * kPath32;
  if (use_fused(m, kv, n)) {
    FusedArgs a = kv->fz;
    a.lw = (const void* const*)m->ftab;
    a.wte = (const uint16_t*)m->wte;
    a.wpe = (const uint16_t*)m->wpe;
    a.lnf_g = (const uint16_t*)m->lnf_g;
    a.lnf_b = (const uint16_t*)m->lnf_b;
    a.p_head = m->p_head;
    a.q8 = m->q8 ? 1 : 0;
    a.L = L;
    a.d = d;
    a.H = H;
    a.M = M;
    a.V = V;
    a.eps = c.ln_eps;
    a.scale = 1.0f / std::sqrt((float)DH);
    a.kc = (const uint16_t*)kv->kc;
    a.vc = (const uint16_t*)kv->vc;
    a.kt = (uint16_t*)kv->kt;
    a.vt = (uint16_t*)kv->vt;
    a.max_ctx = kv->max_ctx;
    a.max_nodes = maxn;
    a.tree = kv->d_tree;
    a.N = n;
    a.P = P;
    a.logits = logits;
    a.plan = kv->fz_plan[(n + 15) / 16];
    a.att_units = (P + kFAttRows - 1) / kFAttRows;
    a.l0 = l0;
    a.x_in = l0 > 0 ? x_in : nullptr;
    HIP_TRY(launch_fused(a, s));
    kv->resid_fused = true;
    kv->last_n = n;
    kv->last_layers = L;
    return SSD_OK;
  }
  if (kv->pass_mode == 2) return fail(SSD_E_UNSUPPORTED, "the persistent pass does not apply to this model, session or tree");
  const int gp = kv->gemm_path;
  const bool q8 = m->q8;
  // pass signals (bf16 models; none for a pass that starts past layer 0,
  // which runs without the prefetcher)
  unsigned long long* sig = f32 || l0 > 0 ? nullptr : kv->d_sig;
  kv->resid_fused = false;
  kv->last_n = n;
  kv->last_layers = L;
  if (l0 > 0) HIP_TRY(hipMemcpyAsync(kv->x, x_in, (size_t)n * d * 4, hipMemcpyDeviceToDevice, s));
  else HIP_TRY(launch_embed(f32, m->wte, m->wpe, d_tok, d_pos, n, d, kv->x, sig, kv->d_xcc0, s));

  // GEMM-input leading dimensions (fp32: row stride; bf16: k-steps)
  const int ld_d = f32 ? d : d / 32, ld_m = f32 ? M : M / 32;
  const size_t pstride = (size_t)maxn * d;
  // fp32 models add residuals inside the GEMM; bf16 models leave split-K
  // partials that the next LayerNorm adds (with the bias)
  const int kind_res = f32 ? EPI_RESID : EPI_PARTIAL;
  const int s_o = resid_splits(m, gp, n, d, d), s_pr = resid_splits(m, gp, n, d, M);
  const size_t kv_layer = (size_t)H * DH;  // elements per K/V row across heads

  int pend_S = 0;               // partials waiting to be added to x
  const void* pend_bias = nullptr;
  for (int l = l0; l < L; ++l) {
    HIP_TRY(launch_ln(f32, kv->x, n, d, kv->part, pend_S, pstride, pend_bias, m->ln1_g[l], m->ln1_b[l], c.ln_eps,
                      kv->act_a, ld_d, sig, kv->d_err, s));
    Epi e{};
    e.sig = sig;
    e.bias = m->b_qkv[l];
    e.N = n;
    e.M = 3 * d;
    e.q = kv->q;
    e.kt = (char*)kv->kt + (size_t)l * kv_layer * maxn * es;
    e.vt = (char*)kv->vt + (size_t)l * kv_layer * maxn * es;
    e.d = d;
    e.H = H;
    e.DH = DH;
    e.max_nodes = maxn;
    HIP_TRY(run_gemm(m, gp, n, EPI_QKV, m->w_qkv[l], f32 ? nullptr : m->p_qkv[l], q8 ? m->s_qkv[l] : nullptr,
                     3 * d, d, kv->act_a, e, s));

    AttnArgs a{};
    a.q = kv->q;
    a.kc = kv->kc ? (const char*)kv->kc + (size_t)l * kv_layer * kv->max_ctx * es : nullptr;
    a.vc = kv->vc ? (const char*)kv->vc + (size_t)l * kv_layer * kv->max_ctx * es : nullptr;
    a.kt = e.kt;
    a.vt = e.vt;
    a.depth = d_dep;
    a.anc_off = d_off;
    a.ancl = d_paths;
    a.path32 = d_path32;
    a.out = kv->act_o;
    a.ldo = ld_d;
    a.part = kv->apart;
    a.S = (P + 63) / 64;
    a.N = n;
    a.P = P;
    a.d = d;
    a.H = H;
    a.max_ctx = kv->max_ctx;
    a.max_nodes = maxn;
    a.scale = 1.0f / std::sqrt((float)DH);
    a.CL = attn_chunk(P, H);
    a.nsplit = attn_nsplit(P, H);
    a.sig = sig;
    a.err = kv->d_err;
    HIP_TRY(launch_attn(f32, DH, a, s));

    Epi eo{};
    eo.sig = sig;
    eo.bias = f32 ? m->b_o[l] : nullptr;
    eo.N = n;
    eo.M = d;
    eo.d = d;
    eo.x = kv->x;
    eo.part = kv->part;
    eo.part_stride = (long long)pstride;
    HIP_TRY(run_gemm(m, gp, n, kind_res, m->w_o[l], f32 ? nullptr : m->p_o[l], q8 ? m->s_o[l] : nullptr, d, d,
                     kv->act_o, eo, s));

    HIP_TRY(launch_ln(f32, kv->x, n, d, kv->part, f32 ? 0 : s_o, pstride, m->b_o[l], m->ln2_g[l], m->ln2_b[l],
                      c.ln_eps, kv->act_a, ld_d, sig, kv->d_err, s));
    Epi ef{};
    ef.sig = sig;
    ef.err = kv->d_err;
    ef.bias = m->b_fc[l];
    ef.N = n;
    ef.M = M;
    ef.d = d;
    ef.out = kv->act_f;
    ef.ldo = ld_m;
    HIP_TRY(run_gemm(m, gp, n, EPI_GELU, m->w_fc[l], f32 ? nullptr : m->p_fc[l], q8 ? m->s_fc[l] : nullptr, M, d,
                     kv->act_a, ef, s));

    Epi ep{};
    ep.sig = sig;
    ep.bias = f32 ? m->b_pr[l] : nullptr;
    ep.N = n;
    ep.M = d;
    ep.d = d;
    ep.x = kv->x;
    ep.part = kv->part;
    ep.part_stride = (long long)pstride;
    HIP_TRY(run_gemm(m, gp, n, kind_res, m->w_pr[l], f32 ? nullptr : m->p_pr[l], q8 ? m->s_pr[l] : nullptr, d, M,
                     kv->act_f, ep, s));
    pend_S = f32 ? 0 : s_pr;
    pend_bias = m->b_pr[l];
  }
  HIP_TRY(launch_ln(f32, kv->x, n, d, kv->part, pend_S, pstride, pend_bias, m->lnf_g, m->lnf_b, c.ln_eps, kv->act_a,
                    ld_d, nullptr, kv->d_err, s));
  Epi eh{};
  eh.bias = nullptr;
  eh.N = n;
  eh.M = V;
  eh.d = d;
  eh.logits = logits;
  eh.ldl = V;
  HIP_TRY(run_gemm(m, gp, n, EPI_LOGITS, m->wte, f32 ? nullptr : m->p_head, m->s_head, V, d, kv->act_a, eh, s));
  return SSD_OK;
}

// The greedy accept right after a pass of n nodes whose staged tree is in
// kv->d_tree: from the persistent pass's per-workgroup LM-head maxima, or by
// reading the logits (one kernel per sub-layer).
static ssd_status enqueue_greedy_after_pass(const ssd_model* m, ssd_kv* kv, int32_t n, bool fused, const float* logits,
                                            int32_t* path, int32_t* path_len, int32_t* next, hipStream_t s) {
  const int maxn = kv->max_nodes;
  const int *tok = kv->d_tree, *dep = kv->d_tree + 2 * maxn, *par = kv->d_tree + 3 * maxn;
  if (fused) {
    HIP_TRY(launch_greedy_from_parts(kv->fz.head_part, kFGroups, n, tok, par, dep, path, path_len, next, s));
  } else {
    HIP_TRY(launch_argmax(logits, n, m->cfg.vocab, kv->d_argmax, kv->d_amwork, s));
    HIP_TRY(launch_greedy_walk(tok, par, dep, n, kv->d_argmax, path, path_len, next, s));
  }
  return SSD_OK;
}

// The eager verification entry points: the pass (from layer l0, see
// enqueue_verify), then with accepted_path set the greedy walk.
static ssd_status verify_entry(const ssd_model* m, ssd_kv* kv, int32_t prefix_len, const int32_t* tree_tokens,
                               const int32_t* parent_idx, int32_t n_nodes, int32_t l0, const float* x_in,
                               float* logits, int32_t* accepted_path, int32_t* path_len, int32_t* next_token,
                               void* stream) {
  int32_t md = 0;
  ssd_status st = check_verify_args(m, kv, prefix_len, tree_tokens, parent_idx, n_nodes, logits, &md);
  if (st != SSD_OK) return st;
  if (l0 < 0 || l0 >= m->cfg.n_layer) return fail(SSD_E_INVALID_ARG, "start_layer outside [0, n_layer)");
  if (l0 > 0 && !x_in) return fail(SSD_E_INVALID_ARG, "null x_in with start_layer > 0");
  hipStream_t s = (hipStream_t)stream;
  char* host = nullptr;
  int slot = -1;
  st = acquire_slot(kv, &host, &slot);
  if (st != SSD_OK) return st;
  const size_t used = fill_stage(host, prefix_len, tree_tokens, parent_idx, n_nodes, kv->max_nodes);
  const bool fused = use_fused(m, kv, n_nodes);
  // (a pass from a later layer runs without the weight prefetcher, whose
  // signal schedule assumes every layer)
  if (l0 == 0) st = start_pass_prefetch(m, kv, n_nodes, fused, kv->gemm_path);
  if (st == SSD_OK) st = enqueue_verify(m, kv, prefix_len, n_nodes, host, used, logits, s, l0, x_in);
  if (st == SSD_OK && accepted_path)
    st = enqueue_greedy_after_pass(m, kv, n_nodes, fused, logits, accepted_path, path_len, next_token, s);
  ssd_status st2 = release_slot(kv, slot, s);
  return st != SSD_OK ? st : st2;
}

extern "C" ssd_status ssd_tree_verify_greedy(const ssd_model* m, ssd_kv* kv, int32_t prefix_len,
                                             const int32_t* tree_tokens, const int32_t* parent_idx, int32_t n_nodes,
                                             float* logits, int32_t* accepted_path, int32_t* path_len,
                                             int32_t* next_token, void* stream) {
  if (!accepted_path || !path_len || !next_token) return fail(SSD_E_INVALID_ARG, "null output");
  return verify_entry(m, kv, prefix_len, tree_tokens, parent_idx, n_nodes, 0, nullptr, logits, accepted_path,
                      path_len, next_token, stream);
}

extern "C" ssd_status ssd_tree_verify(const ssd_model* m, ssd_kv* kv, int32_t prefix_len, const int32_t* tree_tokens,
                                      const int32_t* parent_idx, int32_t n_nodes, float* logits, void* stream) {
  return verify_entry(m, kv, prefix_len, tree_tokens, parent_idx, n_nodes, 0, nullptr, logits, nullptr, nullptr,
                      nullptr, stream);
}

extern "C" ssd_status ssd_tree_verify_from(const ssd_model* m, ssd_kv* kv, int32_t prefix_len,
                                           const int32_t* tree_tokens, const int32_t* parent_idx, int32_t n_nodes,
                                           int32_t start_layer, const float* x_in, float* logits,
                                           int32_t* accepted_path, int32_t* path_len, int32_t* next_token,
                                           void* stream) {
  if (!accepted_path != !path_len || !accepted_path != !next_token)
    return fail(SSD_E_INVALID_ARG, "the greedy outputs must be all set or all NULL");
  return verify_entry(m, kv, prefix_len, tree_tokens, parent_idx, n_nodes, start_layer, x_in, logits, accepted_path,
                      path_len, next_token, stream);
}

static ssd_status capture_pass(const ssd_model* m, ssd_kv* kv, int32_t prefix_len, const int32_t* tree_tokens,
                               const int32_t* parent_idx, int32_t n_nodes, float* logits, int32_t* path,
                               int32_t* path_len, int32_t* next, ssd_graph** out);

extern "C" ssd_status ssd_graph_capture_verify(const ssd_model* m, ssd_kv* kv, int32_t prefix_len,
                                               const int32_t* tree_tokens, const int32_t* parent_idx,
                                               int32_t n_nodes, float* logits, void* stream, ssd_graph** out) {
  (void)stream;
  return capture_pass(m, kv, prefix_len, tree_tokens, parent_idx, n_nodes, logits, nullptr, nullptr, nullptr, out);
}

extern "C" ssd_status ssd_graph_capture_verify_greedy(const ssd_model* m, ssd_kv* kv, int32_t prefix_len,
                                                      const int32_t* tree_tokens, const int32_t* parent_idx,
                                                      int32_t n_nodes, float* logits, int32_t* accepted_path,
                                                      int32_t* path_len, int32_t* next_token, void* stream,
                                                      ssd_graph** out) {
  (void)stream;
  if (!accepted_path || !path_len || !next_token) return fail(SSD_E_INVALID_ARG, "null output");
  return capture_pass(m, kv, prefix_len, tree_tokens, parent_idx, n_nodes, logits, accepted_path, path_len,
                      next_token, out);
}

static ssd_status capture_pass(const ssd_model* m, ssd_kv* kv, int32_t prefix_len, const int32_t* tree_tokens,
                               const int32_t* parent_idx, int32_t n_nodes, float* logits, int32_t* path,
                               int32_t* path_len, int32_t* next, ssd_graph** out) {
  if (!out) return fail(SSD_E_INVALID_ARG, "null output");
  int32_t md = 0;
  ssd_status st = check_verify_args(m, kv, prefix_len, tree_tokens, parent_idx, n_nodes, logits, &md);
  if (st != SSD_OK) return st;
  ssd_graph* g = new ssd_graph();
  g->m = m;
  g->kv = kv;
  g->n = n_nodes;
  g->fused = use_fused(m, kv, n_nodes);
  g->gemm_path = kv->gemm_path;
  hipError_t e = hipHostMalloc((void**)&g->pinned, kv->slot_bytes, hipHostMallocDefault);
  if (e != hipSuccess) {
    delete g;
    return fail(SSD_E_DEVICE, std::string("hipHostMalloc: ") + hipGetErrorString(e));
  }
  const size_t used = fill_stage(g->pinned, prefix_len, tree_tokens, parent_idx, n_nodes, kv->max_nodes);
  // capture on a private stream (the legacy null stream cannot be captured);
  // the graph is later launched on the caller's stream
  hipStream_t cs = nullptr;
  e = hipStreamCreateWithFlags(&cs, hipStreamNonBlocking);
  if (e == hipSuccess) e = hipStreamBeginCapture(cs, hipStreamCaptureModeThreadLocal);
  if (e != hipSuccess) {
    if (cs) (void)hipStreamDestroy(cs);
    ssd_graph_destroy(g);
    return fail(SSD_E_DEVICE, std::string("hipStreamBeginCapture: ") + hipGetErrorString(e));
  }
  st = enqueue_verify(m, kv, prefix_len, n_nodes, g->pinned, used, logits, cs, 0, nullptr);
  if (st == SSD_OK && path) st = enqueue_greedy_after_pass(m, kv, n_nodes, g->fused, logits, path, path_len, next, cs);
  hipGraph_t graph = nullptr;
  e = hipStreamEndCapture(cs, &graph);
  (void)hipStreamDestroy(cs);
  if (st != SSD_OK || e != hipSuccess) {
    if (graph) (void)hipGraphDestroy(graph);
    ssd_graph_destroy(g);
    return st != SSD_OK ? st : fail(SSD_E_DEVICE, std::string("hipStreamEndCapture: ") + hipGetErrorString(e));
  }
  g->graph = graph;
  e = hipGraphInstantiate(&g->exec, graph, nullptr, nullptr, 0);
  if (e != hipSuccess) {
    ssd_graph_destroy(g);
    return fail(SSD_E_DEVICE, std::string("hipGraphInstantiate: ") + hipGetErrorString(e));
  }
  *out = g;
  return SSD_OK;
}

extern "C" ssd_status ssd_graph_launch(ssd_graph* g, void* stream) {
  if (!g || !g->exec) return fail(SSD_E_INVALID_ARG, "null graph");
  const ssd_status st = start_pass_prefetch(g->m, g->kv, g->n, g->fused, g->gemm_path);
  if (st != SSD_OK) return st;
  HIP_TRY(hipGraphLaunch(g->exec, (hipStream_t)stream));
  g->kv->resid_fused = g->fused;
  g->kv->last_n = g->n;
  g->kv->last_layers = g->m->cfg.n_layer;
  return SSD_OK;
}

extern "C" void ssd_graph_destroy(ssd_graph* g) {
  if (!g) return;
  if (g->exec) (void)hipGraphExecDestroy(g->exec);
  if (g->graph) (void)hipGraphDestroy(g->graph);
  if (g->pinned) (void)hipHostFree(g->pinned);
  delete g;
}

extern "C" ssd_status ssd_launch_gemm(const ssd_model* m, ssd_kv* kv, int32_t which, int32_t layer, int32_t n_nodes,
                                      void* stream) {
  if (!m || !kv) return fail(SSD_E_INVALID_ARG, "null argument");
  if (kv->m != m && !same_shape_prefix(m->cfg, kv->m->cfg))
    return fail(SSD_E_INVALID_ARG, "the model's shape differs from the session's");
  const ssd_config& c = m->cfg;
  if (which < 0 || which > 3 || layer < 0 || layer >= c.n_layer) return fail(SSD_E_INVALID_ARG, "bad matrix id");
  if (n_nodes <= 0 || n_nodes > kv->max_nodes) return fail(SSD_E_CAPACITY, "n_nodes outside the session");
  const int d = c.d_model, M = c.d_mlp, es = m->f32 ? 4 : 2;
  // outputs land in the session's own workspaces (q and tree scratch, split-K
  // partials or x, the MLP activation buffer)
  Epi e{};
  e.N = n_nodes;
  e.d = d;
  e.H = c.n_head;
  e.DH = m->dh;
  e.max_nodes = kv->max_nodes;
  e.x = kv->x;
  e.part = kv->part;
  e.part_stride = (long long)kv->max_nodes * d;
  const int kind_res = m->f32 ? EPI_RESID : EPI_PARTIAL;
  const void *Wraw = nullptr, *Wp = nullptr, *act = kv->act_a;
  const float* wscale = nullptr;
  int rows = d, K = d, lda = d, kind = kind_res;
  switch (which) {
    case 0:
      kind = EPI_QKV; rows = 3 * d; Wraw = m->w_qkv[layer]; e.bias = m->b_qkv[layer]; e.q = kv->q;
      e.kt = (char*)kv->kt + (size_t)layer * c.n_head * m->dh * kv->max_nodes * es;
      e.vt = (char*)kv->vt + (size_t)layer * c.n_head * m->dh * kv->max_nodes * es;
      if (!m->f32) Wp = m->p_qkv[layer];
      if (m->q8) wscale = m->s_qkv[layer];
      break;
    case 1:
      Wraw = m->w_o[layer]; act = kv->act_o; if (m->f32) e.bias = m->b_o[layer];
      if (!m->f32) Wp = m->p_o[layer];
      if (m->q8) wscale = m->s_o[layer];
      break;
    case 2:
      kind = EPI_GELU; rows = M; Wraw = m->w_fc[layer]; e.bias = m->b_fc[layer]; e.out = kv->act_f;
      e.ldo = m->f32 ? M : M / 32;
      if (!m->f32) Wp = m->p_fc[layer];
      if (m->q8) wscale = m->s_fc[layer];
      break;
    default:
      K = M; lda = M; Wraw = m->w_pr[layer]; act = kv->act_f; if (m->f32) e.bias = m->b_pr[layer];
      if (!m->f32) Wp = m->p_pr[layer];
      if (m->q8) wscale = m->s_pr[layer];
      break;
  }
  e.M = rows;
  (void)lda;
  HIP_TRY(run_gemm(m, kv->gemm_path, n_nodes, kind, Wraw, Wp, wscale, rows, K, act, e, (hipStream_t)stream));
  return SSD_OK;
}

// ------------------------------------------------------------------ top-k

extern "C" ssd_status ssd_topk(ssd_kv* kv, const float* logits, int32_t n_rows, int32_t k, int32_t* idx, float* val,
                               float* lse, void* stream) {
  if (!kv || !logits || !idx || !val) return fail(SSD_E_INVALID_ARG, "null argument");
  if (k < 1 || k > kTopKMax) return fail(SSD_E_INVALID_ARG, "k outside [1, 8]");
  if (n_rows < 1 || n_rows > kv->max_nodes) return fail(SSD_E_CAPACITY, "n_rows outside [1, max_nodes]");
  hipStream_t s = (hipStream_t)stream;
  HIP_TRY(launch_topk(logits, n_rows, kv->m->cfg.vocab, k, idx, val, lse, kv->d_amwork, s));
  return SSD_OK;
}

// ------------------------------------------------------------------ accept

// accept-mode rules shared by both accept entry points
static ssd_status check_accept_mode(const ssd_tree* tree, const float* draft_probs) {
  const int mode = tree->mode;
  if (mode != SSD_ACCEPT_GREEDY && mode != SSD_ACCEPT_SAMPLE_WOR && mode != SSD_ACCEPT_SAMPLE_IID &&
      mode != SSD_ACCEPT_SAMPLE_DET && mode != SSD_ACCEPT_SAMPLE_CDF)
    return fail(SSD_E_INVALID_ARG, "unknown accept mode");
  const bool drawn = mode == SSD_ACCEPT_SAMPLE_WOR || mode == SSD_ACCEPT_SAMPLE_IID;
  if (drawn && !draft_probs) return fail(SSD_E_INVALID_ARG, "draft_probs required when siblings were drawn");
  if (!drawn && draft_probs) return fail(SSD_E_INVALID_ARG, "draft_probs must be NULL for this accept mode");
  if (mode != SSD_ACCEPT_GREEDY && !(tree->temperature > 0.f))
    return fail(SSD_E_INVALID_ARG, "temperature must be positive");
  if (tree->top_k < 0) return fail(SSD_E_INVALID_ARG, "top_k must be >= 0");
  if (mode != SSD_ACCEPT_GREEDY && tree->vocab > kSampleMaxVocab)
    return fail(SSD_E_CAPACITY, "vocab above 131072 (the sampling walk's limit)");
  return SSD_OK;
}

extern "C" ssd_status ssd_tree_accept(ssd_kv* kv, const ssd_tree* tree, const float* draft_probs,
                                      const float* oracle_logits, uint64_t rng_seed, int32_t* accepted_path,
                                      int32_t* path_len, int32_t* next_token, void* stream) {
  if (!kv || !tree || !oracle_logits || !accepted_path || !path_len || !next_token)
    return fail(SSD_E_INVALID_ARG, "null argument");
  const int n = tree->n_nodes, V = tree->vocab;
  if (n <= 0 || V <= 0) return fail(SSD_E_INVALID_ARG, "n_nodes and vocab must be positive");
  if (n > kv->max_nodes) return fail(SSD_E_CAPACITY, "n_nodes above the session's max_nodes");
  if (V > kv->m->cfg.vocab) return fail(SSD_E_CAPACITY, "vocab above the model's vocab");
  ssd_status st = check_accept_mode(tree, draft_probs);
  if (st != SSD_OK) return st;
  const bool greedy = tree->mode == SSD_ACCEPT_GREEDY;
  int32_t md = 0;
  st = ssd_validate_tree(tree->tokens, tree->parent_idx, n, V, &md);
  if (st != SSD_OK) return st;
  hipStream_t s = (hipStream_t)stream;
  char* host = nullptr;
  int slot = -1;
  st = acquire_slot(kv, &host, &slot);
  if (st != SSD_OK) return st;
  int32_t* t = (int32_t*)host;
  int32_t* par = t + n;
  int32_t* dep = par + n;
  for (int i = 0; i < n; ++i) {
    t[i] = tree->tokens[i];
    par[i] = tree->parent_idx[i];
    dep[i] = i == 0 ? 0 : dep[par[i]] + 1;
  }
  int* dt = kv->d_accept_tree;
  HIP_TRY(hipMemcpyAsync(dt, host, (size_t)3 * n * 4, hipMemcpyHostToDevice, s));
  if (greedy) {
    HIP_TRY(launch_argmax(oracle_logits, n, V, kv->d_argmax, kv->d_amwork, s));
    HIP_TRY(launch_greedy_walk(dt, dt + n, dt + 2 * n, n, kv->d_argmax, accepted_path, path_len, next_token, s));
  } else {
    HIP_TRY(launch_sample_accept(dt, dt + n, n, V, oracle_logits, draft_probs, (double)tree->temperature, rng_seed,
                                 (int)tree->mode, tree->top_k, kv->d_sw, kv->d_err, accepted_path, path_len,
                                 next_token, s));
  }
  return release_slot(kv, slot, s);
}

// ------------------------------------------------------------------ accept without allocation
//
// For callers that cannot allocate device memory (code under HIP graph
// capture, tight serving loops, harnesses that forbid hipMalloc): the accept
// walk with its scratch in one file-scope device array instead of a
// session's workspace.  The array holds the staged tree, the argmax partials
// and results, and the sampling walk's exchange area.  The argmax kernels
// write what they later read; the exchange area starts zeroed (as the array
// does when the module loads) and the sampler keeps it consistent itself
// (an epoch raised by every call), so nothing needs clearing between calls.
// Each device gets its own copy of the array at its own address, fetched once
// per device with hipGetSymbolAddress; every call on a device shares it, so
// calls that overlap on one device (two streams, or two host threads) race.
constexpr int kNaMaxNodes = 256;
constexpr int kNaMaxVocab = 65536;
constexpr size_t kNaTreeOfs = 0;                                  // tokens, parents, depth: int32[3][kNaMaxNodes]
constexpr size_t kNaArgOfs = 4096;                                // argmax results: int32[kNaMaxNodes]
constexpr size_t kNaWorkOfs = 8192;                               // argmax partials
constexpr size_t kNaWorkBytes = (size_t)kNaMaxNodes * ((kNaMaxVocab + 2047) / 2048) * 8;
constexpr size_t kNaSwOfs = kNaWorkOfs + kNaWorkBytes;            // the sampling walk's exchange area
constexpr size_t kNaScratchBytes = kNaSwOfs + kSampleWorkBytes;
static_assert(kNaScratchBytes <= (2u << 20), "the no-allocation scratch is at most 2 MiB per device");
static __device__ __align__(256) unsigned char scratch[kNaScratchBytes];

// the tree travels in the kernel's arguments (no host-to-device copy)
struct NaTree {
  int32_t tokens[kNaMaxNodes];
  int32_t parents[kNaMaxNodes];
  int32_t n;
};

// tokens, parents and depths into the scratch's tree rows (validated on the host)
__global__ __launch_bounds__(256) void na_tree_kernel(NaTree t, int32_t* out) {
  const int n = t.n;
  for (int i = threadIdx.x; i < n; i += blockDim.x) {
    out[i] = t.tokens[i];
    out[kNaMaxNodes + i] = t.parents[i];
  }
  if (threadIdx.x == 0) {
    int32_t* dep = out + 2 * kNaMaxNodes;
    dep[0] = 0;
    for (int i = 1; i < n; ++i) dep[i] = dep[t.parents[i]] + 1;
  }
}

static std::mutex g_na_mu;
static void* g_na_ptr[64] = {};

// this device's address of `scratch` (looked up once per device)
static ssd_status na_scratch(unsigned char** out) {
  int dev = 0;
  HIP_TRY(hipGetDevice(&dev));
  if (dev < 0 || dev >= 64) return fail(SSD_E_DEVICE, "device index beyond 63");
  std::lock_guard<std::mutex> lk(g_na_mu);
  if (!g_na_ptr[dev]) {
    void* p = nullptr;
    const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return fail(SSD_E_DEVICE, std::string("hipGetSymbolAddress(scratch): ") + hipGetErrorString(e));
    g_na_ptr[dev] = p;
  }
  *out = (unsigned char*)g_na_ptr[dev];
  return SSD_OK;
}

extern "C" ssd_status ssd_tree_accept_noalloc(const ssd_tree* tree, const float* draft_probs,
                                              const float* oracle_logits, uint64_t rng_seed, int32_t* accepted_path,
                                              int32_t* path_len, int32_t* next_token, void* stream) {
  if (!tree || !oracle_logits || !accepted_path || !path_len || !next_token)
    return fail(SSD_E_INVALID_ARG, "null argument");
  const int n = tree->n_nodes, V = tree->vocab;
  if (n <= 0 || V <= 0) return fail(SSD_E_INVALID_ARG, "n_nodes and vocab must be positive");
  if (n > kNaMaxNodes) return fail(SSD_E_CAPACITY, "n_nodes above 256 (the no-allocation accept's limit)");
  if (V > kNaMaxVocab) return fail(SSD_E_CAPACITY, "vocab above 65536 (the no-allocation accept's limit)");
  ssd_status st = check_accept_mode(tree, draft_probs);
  if (st != SSD_OK) return st;
  const bool greedy = tree->mode == SSD_ACCEPT_GREEDY;
  if (argmax_work_bytes(n, V) > kNaWorkBytes) return fail(SSD_E_CAPACITY, "argmax partials exceed the scratch");
  int32_t md = 0;
  st = ssd_validate_tree(tree->tokens, tree->parent_idx, n, V, &md);
  if (st != SSD_OK) return st;
  unsigned char* base = nullptr;
  st = na_scratch(&base);
  if (st != SSD_OK) return st;
  NaTree t{};
  t.n = n;
  for (int i = 0; i < n; ++i) {
    t.tokens[i] = tree->tokens[i];
    t.parents[i] = tree->parent_idx[i];
  }
  hipStream_t s = (hipStream_t)stream;
  int32_t* dt = (int32_t*)(base + kNaTreeOfs);
  na_tree_kernel<<<1, 256, 0, s>>>(t, dt);
  HIP_TRY(hipGetLastError());
  if (greedy) {
    int32_t* g = (int32_t*)(base + kNaArgOfs);
    HIP_TRY(launch_argmax(oracle_logits, n, V, g, base + kNaWorkOfs, s));
    HIP_TRY(launch_greedy_walk(dt, dt + kNaMaxNodes, dt + 2 * kNaMaxNodes, n, g, accepted_path, path_len, next_token,
                               s));
  } else {
    HIP_TRY(launch_sample_accept(dt, dt + kNaMaxNodes, n, V, oracle_logits, draft_probs, (double)tree->temperature,
                                 rng_seed, (int)tree->mode, tree->top_k, base + kNaSwOfs, nullptr, accepted_path,
                                 path_len, next_token, s));
  }
  return SSD_OK;
}

// ------------------------------------------------------------------ commit

extern "C" ssd_status ssd_kv_commit(ssd_kv* kv, int32_t prefix_len, const int32_t* accepted_path,
                                    const int32_t* path_len, void* stream) {
  if (!kv || !accepted_path || !path_len) return fail(SSD_E_INVALID_ARG, "null argument");
  if (prefix_len < 0 || prefix_len > kv->max_ctx) return fail(SSD_E_CAPACITY, "prefix_len outside the cache");
  if (!kv->kc) return fail(SSD_E_CAPACITY, "session has no cache");
  const ssd_model* m = kv->m;
  HIP_TRY(launch_commit(m->f32 ? 1 : 0, kv->kc, kv->vc, kv->kt, kv->vt, m->cfg.n_layer * m->cfg.n_head, kv->max_ctx,
                        kv->max_nodes, m->dh, prefix_len, accepted_path, path_len, kv->d_err, (hipStream_t)stream));
  return SSD_OK;
}

extern "C" ssd_status ssd_kv_error_count(ssd_kv* kv, void* stream, uint32_t* count) {
  if (!kv || !count) return fail(SSD_E_INVALID_ARG, "null argument");
  unsigned h = 0;
  HIP_TRY(hipMemcpyAsync(&h, kv->d_err, 4, hipMemcpyDeviceToHost, (hipStream_t)stream));
  HIP_TRY(hipStreamSynchronize((hipStream_t)stream));
  *count = h;
  return SSD_OK;
}

// ------------------------------------------------------------------ 8-bit weights, read back

extern "C" ssd_status ssd_model_q8_matrix(const ssd_model* m, int32_t which, int32_t layer, int8_t* codes,
                                          float* scales) {
  if (!m || !codes || !scales) return fail(SSD_E_INVALID_ARG, "null argument");
  if (!m->q8) return fail(SSD_E_INVALID_ARG, "the model has no 8-bit weights");
  const ssd_config& c = m->cfg;
  if (which < 0 || which > 4 || (which < 4 && (layer < 0 || layer >= c.n_layer)))
    return fail(SSD_E_INVALID_ARG, "bad matrix id or layer");
  const int d = c.d_model, M = c.d_mlp;
  const int rows[5] = {3 * d, d, M, d, c.vocab}, Ks[5] = {d, d, d, M, d};
  const void* frag[5] = {nullptr, nullptr, nullptr, nullptr, m->p_head};
  const float* sc[5] = {nullptr, nullptr, nullptr, nullptr, m->s_head};
  if (which < 4) {
    frag[which] = (which == 0 ? m->p_qkv : which == 1 ? m->p_o : which == 2 ? m->p_fc : m->p_pr)[layer];
    sc[which] = (which == 0 ? m->s_qkv : which == 1 ? m->s_o : which == 2 ? m->s_fc : m->s_pr)[layer];
  }
  const int R = rows[which], K = Ks[which], KC = K / 32;
  std::vector<uint8_t> f(packed_q8_bytes(R, K));
  HIP_TRY(hipDeviceSynchronize());
  HIP_TRY(hipMemcpy(f.data(), frag[which], f.size(), hipMemcpyDeviceToHost));
  HIP_TRY(hipMemcpy(scales, sc[which], (size_t)R * 4, hipMemcpyDeviceToHost));
  // fragment (rb, kc), lane l, byte j: row 16 rb + l % 16, k = 32 kc + 8 (l / 16) + j
  for (int r = 0; r < R; ++r)
    for (int k = 0; k < K; ++k) {
      const int rb = r / 16, kc = k / 32, lane = (r % 16) + 16 * ((k % 32) / 8);
      codes[(size_t)r * K + k] = (int8_t)((int)f[(((size_t)rb * KC + kc) * 64 + lane) * 8 + k % 8] - 128);
    }
  return SSD_OK;
}

// ------------------------------------------------------------------ host uniforms

// Philox4x64-10 (Salmon, Moraes, Dror, Shaw, SC'11): ten rounds of two 64x64
// multiplies with the published multipliers, the key bumped by the published
// Weyl constants between rounds; the same generator the accept kernels run.
extern "C" double ssd_uniform(uint64_t seed, uint64_t stream, uint64_t counter) {
  const uint64_t M0 = 0xD2E7470EE14C6C93ull, M1 = 0xCA5A826395121157ull;
  const uint64_t W0 = 0x9E3779B97F4A7C15ull, W1 = 0xBB67AE8584CAA73Bull;
  uint64_t c0 = counter, c1 = 0, c2 = 0, c3 = 0, k0 = seed, k1 = stream;
  for (int r = 0; r < 10; ++r) {
    if (r) {
      k0 += W0;
      k1 += W1;
    }
    const unsigned __int128 p0 = (unsigned __int128)M0 * c0, p1 = (unsigned __int128)M1 * c2;
    const uint64_t n0 = (uint64_t)(p1 >> 64) ^ c1 ^ k0, n2 = (uint64_t)(p0 >> 64) ^ c3 ^ k1;
    c1 = (uint64_t)p1;
    c3 = (uint64_t)p0;
    c0 = n0;
    c2 = n2;
  }
  return (double)(c0 >> 11) * 0x1.0p-53;
}

// ------------------------------------------------------------------ inverse-CDF picks

extern "C" ssd_status ssd_cdf_pick(ssd_kv* kv, const float* logits, int32_t n_rows, int32_t vocab, float temperature,
                                   int32_t n_queries, const int32_t* rows, const double* uniforms, int32_t* tokens,
                                   void* stream) {
  if (!kv || !logits || !rows || !uniforms || !tokens) return fail(SSD_E_INVALID_ARG, "null argument");
  if (n_rows < 1 || n_rows > kv->max_nodes) return fail(SSD_E_CAPACITY, "n_rows outside [1, max_nodes]");
  if (vocab < 1 || vocab > kv->m->cfg.vocab) return fail(SSD_E_INVALID_ARG, "vocab outside [1, the model's vocab]");
  if (n_queries < 1 || n_queries > kMaxPicks) return fail(SSD_E_INVALID_ARG, "n_queries outside [1, 64]");
  if (!(temperature > 0.f)) return fail(SSD_E_INVALID_ARG, "temperature must be positive");
  CdfPickArgs a{};
  a.logits = logits;
  a.V = vocab;
  a.n = n_queries;
  a.T = temperature;
  a.out = tokens;
  for (int q = 0; q < n_queries; ++q) {
    if (rows[q] < 0 || rows[q] >= n_rows) return fail(SSD_E_INVALID_ARG, "row outside [0, n_rows)");
    if (!(uniforms[q] >= 0.0 && uniforms[q] < 1.0)) return fail(SSD_E_INVALID_ARG, "uniform outside [0, 1)");
    a.rows[q] = rows[q];
    a.U[q] = uniforms[q];
  }
  HIP_TRY(launch_cdf_pick(a, (hipStream_t)stream));
  return SSD_OK;
}

// ------------------------------------------------------------------ draft work reused by the oracle pass

// Block i copies node src_rows[i]'s tree K/V rows of the first LH / H layers
// and its residual row into the destination's slot i.
constexpr int kMaxReuse = 256;
struct ReuseArgs {
  const unsigned char *ks, *vs;
  unsigned char *kd, *vd;
  const float* xs;
  float* xd;
  int LH, src_rows, dst_rows, row_bytes, d;
  int rows[kMaxReuse];
};

__global__ __launch_bounds__(256) void tree_reuse_kernel(ReuseArgs a) {
  const int i = blockIdx.x, sr = a.rows[i];
  const int per = a.row_bytes / 16;  // 16-byte pieces of a K or V row
  for (int t = threadIdx.x; t < a.LH * per; t += 256) {
    const int lh = t / per, c = t - lh * per;
    const size_t so = ((size_t)lh * a.src_rows + sr) * a.row_bytes + 16 * c;
    const size_t dof = ((size_t)lh * a.dst_rows + i) * a.row_bytes + 16 * c;
    *(uint4*)(a.kd + dof) = *(const uint4*)(a.ks + so);
    *(uint4*)(a.vd + dof) = *(const uint4*)(a.vs + so);
  }
  for (int t = threadIdx.x; t < a.d; t += 256) a.xd[(size_t)i * a.d + t] = a.xs[(size_t)sr * a.d + t];
}

extern "C" ssd_status ssd_tree_reuse(const ssd_kv* src, ssd_kv* dst, int32_t n, const int32_t* src_rows, float* x_out,
                                     void* stream) {
  if (!src || !dst || !src_rows || !x_out) return fail(SSD_E_INVALID_ARG, "null argument");
  if (src == dst) return fail(SSD_E_INVALID_ARG, "source and destination sessions must differ");
  const ssd_config &cs = src->m->cfg, &cd = dst->m->cfg;
  if (!same_shape_prefix(cs, cd)) return fail(SSD_E_INVALID_ARG, "the source model is not a layer prefix of the destination's");
  if (n < 1 || n > kMaxReuse || n > dst->max_nodes) return fail(SSD_E_CAPACITY, "n outside [1, min(256, max_nodes)]");
  if (src->last_layers < 1 || src->last_layers > cd.n_layer)
    return fail(SSD_E_INVALID_ARG, "no pass of a layer prefix of the destination's model ran on the source session");
  ReuseArgs a{};
  for (int i = 0; i < n; ++i) {
    if (src_rows[i] < 0 || src_rows[i] >= src->last_n)
      return fail(SSD_E_INVALID_ARG, "a source row outside the source session's last pass");
    a.rows[i] = src_rows[i];
  }
  const int es = cs.dtype == SSD_F32 ? 4 : 2, dh = cs.d_model / cs.n_head;
  a.ks = (const unsigned char*)src->kt;
  a.vs = (const unsigned char*)src->vt;
  a.kd = (unsigned char*)dst->kt;
  a.vd = (unsigned char*)dst->vt;
  a.LH = src->last_layers * cs.n_head;
  a.src_rows = src->max_nodes;
  a.dst_rows = dst->max_nodes;
  a.row_bytes = dh * es;
  a.d = cs.d_model;
  a.xs = src->resid_fused ? src->fz.xr : src->x;  // (the persistent pass: XCD 0's copy, rows of kFMaxN)
  a.xd = x_out;
  tree_reuse_kernel<<<n, 256, 0, (hipStream_t)stream>>>(a);
  HIP_TRY(hipGetLastError());
  return SSD_OK;
}
