// Internal declarations shared by the HIP kernels (kernels.hip) and the host
// runtime (runtime.hip) of libssd.  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ssd {

// Epilogues of the skinny GEMM Y[n][o] = sum_k A[n][k] W[o][k].
enum EpiKind : int {
  EPI_QKV = 0,    // +bias; o < d -> q (fp32); d <= o < 2d -> K scratch; 2d <= o -> V scratch
  EPI_RESID = 1,  // x[n][o] += y + bias[o]
  EPI_GELU = 2,   // out[n][o] = gelu_tanh(y + bias[o])  (storage of the activation buffer)
  EPI_LOGITS = 3  // logits[n][o] = y
};

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
  int ldo;
  long long out_plane;  // bf16 models: elements from the hi plane to the lo plane
  // EPI_LOGITS
  float* logits;
  long long ldl;
};

struct AttnArgs {
  const float* q;    // [N][d]
  const void* kc;    // cache, this layer: [H][max_ctx][DH]
  const void* vc;
  const void* kt;    // tree scratch, this layer: [H][max_nodes][DH]
  const void* vt;
  const uint64_t* anc;  // [N][W]
  float* part;       // [H][NS][N][DH + 2]
  int N, P, d, H, max_ctx, max_nodes, W, S, NS;
  float scale;
};

// ---- launchers (kernels.hip); all enqueue on `s` and return the launch status
hipError_t launch_embed(int f32, const void* wte, const void* wpe, const int* tokens, const int* pos, int N, int d,
                        float* x, hipStream_t s);
// bf16 activation buffers hold a hi plane and, `plane` elements later, a lo plane
hipError_t launch_ln(int f32, const float* x, int N, int d, const void* g, const void* b, float eps, void* a,
                     int lda, size_t plane, hipStream_t s);
hipError_t launch_gemm_f32(int kind, const float* W, int M, int K, const float* act, int lda, const Epi& ep,
                           hipStream_t s);
// Wp: weights packed in 16x32 bf16 fragments (see pack); act: bf16 hi plane [>= 16*NT rows][lda],
// lo plane `plane` elements later
hipError_t launch_gemm_mfma(int kind, const void* Wp, int M, int K, const uint16_t* act, int lda, size_t plane,
                            const Epi& ep, hipStream_t s);
hipError_t launch_gemm_vec(int kind, const void* Wp, int M, int K, const uint16_t* act, int lda, size_t plane,
                           const Epi& ep, hipStream_t s);
hipError_t launch_attn(int f32, int DH, const AttnArgs& a, hipStream_t s);
hipError_t launch_attn_combine(int f32, int DH, const float* part, int NS, int N, int H, int d, void* out, int ldo,
                               size_t plane, hipStream_t s);
hipError_t launch_pack_bf16(const uint16_t* W, int M, int K, void* out, hipStream_t s);
size_t packed_bytes(int M, int K);
hipError_t launch_argmax(const float* logits, int N, int V, int* g, hipStream_t s);
hipError_t launch_greedy_walk(const int* tokens, const int* parents, const int* depth, int N, const int* g,
                              int* path, int* path_len, int* next, hipStream_t s);
hipError_t launch_sample_accept(const int* tokens, const int* parents, int N, int V, const float* logits,
                                const float* draft, double temperature, uint64_t seed, int wor, double* r, double* p,
                                double* qq, int* path, int* path_len, int* next, hipStream_t s);
hipError_t launch_commit(int f32, void* kc, void* vc, const void* kt, const void* vt, int LH, int max_ctx,
                         int max_nodes, int DH, int P, const int* path, const int* path_len, unsigned* err,
                         hipStream_t s);

}  // namespace ssd
