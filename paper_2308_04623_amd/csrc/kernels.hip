// HIP kernels of libssd for CDNA4 (gfx950): one decoder pass over a token
// tree (Sec. 3.1 of Spector & Re, arXiv 2308.04623), the accept/reject walk
// (Sec. 2.3) and the KV commit.
//
// Data layout (HBM):
//   x        fp32 [N][d]         residual stream
//   q        fp32 [N][d]         queries of the current layer
//   act_*    bf16 (or fp32 for fp32 models) [Npad][d or d_mlp], GEMM inputs
//   K/V      storage type [L][H][rows][DH] (cache rows: positions; scratch rows: nodes)
//   packed W 16x32 bf16 fragments; fragment (rb, kc) holds rows 16rb.., k 32kc..,
//            lane l's 16 bytes = W[16rb + l%16][32kc + 8(l/16) .. +8], fragments
//            ordered rb-major so one wave streams 1 KB contiguous per load.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "ssd_internal.h"

namespace ssd {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));

// ------------------------------------------------------------------ helpers

__device__ __forceinline__ float bf2f(uint16_t h) { return __uint_as_float((uint32_t)h << 16); }

// float -> bfloat16, round to nearest even
__device__ __forceinline__ uint16_t f2bf(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)0x7fc0;
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

template <typename T> __device__ __forceinline__ float ldT(const T* p, size_t i);
template <> __device__ __forceinline__ float ldT<float>(const float* p, size_t i) { return p[i]; }
template <> __device__ __forceinline__ float ldT<uint16_t>(const uint16_t* p, size_t i) { return bf2f(p[i]); }

template <typename T> __device__ __forceinline__ void stT(T* p, size_t i, float v);
template <> __device__ __forceinline__ void stT<float>(float* p, size_t i, float v) { p[i] = v; }
template <> __device__ __forceinline__ void stT<uint16_t>(uint16_t* p, size_t i, float v) { p[i] = f2bf(v); }

// GEMM inputs of bf16 models are stored as two bf16 planes, hi = bf16(v) and
// lo = bf16(v - hi), `plane` elements apart; the GEMMs multiply both, which
// keeps about 16 significant bits of every activation.
template <typename T> __device__ __forceinline__ void st_act(T* p, size_t i, size_t plane, float v);
template <> __device__ __forceinline__ void st_act<float>(float* p, size_t i, size_t, float v) { p[i] = v; }
template <> __device__ __forceinline__ void st_act<uint16_t>(uint16_t* p, size_t i, size_t plane, float v) {
  const uint16_t hi = f2bf(v);
  p[i] = hi;
  p[i + plane] = f2bf(v - bf2f(hi));
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}

// sum over a 256-thread block, identical result in every thread, fixed order
__device__ __forceinline__ float block_sum256(float v, float* red4) {
  v = wave_sum(v);
  const int w = threadIdx.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red4[w] = v;
  __syncthreads();
  return (red4[0] + red4[1]) + (red4[2] + red4[3]);
}

__device__ __forceinline__ float gelu_tanh(float x) {
  const float c = 0.7978845608028654f;  // sqrt(2/pi)
  return 0.5f * x * (1.0f + tanhf(c * (x + 0.044715f * x * x * x)));
}

// ------------------------------------------------------------------ embed

template <typename T>
__global__ __launch_bounds__(256) void embed_kernel(const T* __restrict__ wte, const T* __restrict__ wpe,
                                                    const int* __restrict__ tokens, const int* __restrict__ pos,
                                                    int d, float* __restrict__ x) {
  const int n = blockIdx.x;
  const size_t t = (size_t)tokens[n] * d, p = (size_t)pos[n] * d;
  for (int k = threadIdx.x; k < d; k += blockDim.x) x[(size_t)n * d + k] = ldT(wte, t + k) + ldT(wpe, p + k);
}

hipError_t launch_embed(int f32, const void* wte, const void* wpe, const int* tokens, const int* pos, int N, int d,
                        float* x, hipStream_t s) {
  if (f32)
    embed_kernel<float><<<N, 256, 0, s>>>((const float*)wte, (const float*)wpe, tokens, pos, d, x);
  else
    embed_kernel<uint16_t><<<N, 256, 0, s>>>((const uint16_t*)wte, (const uint16_t*)wpe, tokens, pos, d, x);
  return hipGetLastError();
}

// ------------------------------------------------------------------ LayerNorm

// a[n] = (x[n] - mean) / sqrt(var + eps) * g + b   (biased variance, fp32)
template <typename T, typename OUT>
__global__ __launch_bounds__(256) void ln_kernel(const float* __restrict__ x, int d, const T* __restrict__ g,
                                                 const T* __restrict__ b, float eps, OUT* __restrict__ a, int lda,
                                                 size_t plane) {
  __shared__ float red[4];
  const int n = blockIdx.x;
  const float* xr = x + (size_t)n * d;
  float s = 0.f;
  for (int k = threadIdx.x; k < d; k += 256) s += xr[k];
  const float mean = block_sum256(s, red) / d;
  float v = 0.f;
  for (int k = threadIdx.x; k < d; k += 256) {
    const float t = xr[k] - mean;
    v += t * t;
  }
  const float var = block_sum256(v, red) / d;
  const float den = sqrtf(var + eps);
  for (int k = threadIdx.x; k < d; k += 256)
    st_act(a, (size_t)n * lda + k, plane, (xr[k] - mean) / den * ldT(g, k) + ldT(b, k));
}

hipError_t launch_ln(int f32, const float* x, int N, int d, const void* g, const void* b, float eps, void* a,
                     int lda, size_t plane, hipStream_t s) {
  if (f32)
    ln_kernel<float, float><<<N, 256, 0, s>>>(x, d, (const float*)g, (const float*)b, eps, (float*)a, lda, 0);
  else
    ln_kernel<uint16_t, uint16_t><<<N, 256, 0, s>>>(x, d, (const uint16_t*)g, (const uint16_t*)b, eps,
                                                     (uint16_t*)a, lda, plane);
  return hipGetLastError();
}

// ------------------------------------------------------------------ GEMM epilogues

template <typename T, int KIND>
__device__ __forceinline__ void epilogue(const Epi& e, int n, int o, float acc) {
  const float y = acc + (e.bias ? ldT((const T*)e.bias, o) : 0.f);
  const int nn = e.node0 + n;
  if (KIND == EPI_QKV) {
    if (o < e.d) {
      e.q[(size_t)nn * e.d + o] = y;
    } else {
      const int oo = o < 2 * e.d ? o - e.d : o - 2 * e.d;
      const int h = oo / e.DH, j = oo - h * e.DH;
      T* dst = (T*)(o < 2 * e.d ? e.kt : e.vt);
      stT(dst, ((size_t)h * e.max_nodes + nn) * e.DH + j, y);
    }
  } else if (KIND == EPI_RESID) {
    e.x[(size_t)nn * e.d + o] += y;
  } else if (KIND == EPI_GELU) {
    st_act((T*)e.out, (size_t)nn * e.ldo + o, (size_t)e.out_plane, gelu_tanh(y));
  } else {
    e.logits[(size_t)nn * e.ldl + o] = acc;
  }
}

// ------------------------------------------------------------------ GEMM, fp32 models

// One thread per (node, output row); only used for the small fp32 model.
template <int KIND>
__global__ __launch_bounds__(256) void gemm_f32_kernel(const float* __restrict__ W, int M, int K,
                                                       const float* __restrict__ act, int lda, Epi ep) {
  const int o = blockIdx.x * 256 + threadIdx.x, n = blockIdx.y;
  if (o >= M) return;
  const float* wr = W + (size_t)o * K;
  const float* ar = act + (size_t)n * lda;
  float acc = 0.f;
  for (int k = 0; k < K; ++k) acc = fmaf(ar[k], wr[k], acc);
  epilogue<float, KIND>(ep, n, o, acc);
}

hipError_t launch_gemm_f32(int kind, const float* W, int M, int K, const float* act, int lda, const Epi& ep,
                           hipStream_t s) {
  dim3 grid((M + 255) / 256, ep.N);
  switch (kind) {
    case EPI_QKV: gemm_f32_kernel<EPI_QKV><<<grid, 256, 0, s>>>(W, M, K, act, lda, ep); break;
    case EPI_RESID: gemm_f32_kernel<EPI_RESID><<<grid, 256, 0, s>>>(W, M, K, act, lda, ep); break;
    case EPI_GELU: gemm_f32_kernel<EPI_GELU><<<grid, 256, 0, s>>>(W, M, K, act, lda, ep); break;
    default: gemm_f32_kernel<EPI_LOGITS><<<grid, 256, 0, s>>>(W, M, K, act, lda, ep); break;
  }
  return hipGetLastError();
}

// ------------------------------------------------------------------ weight packing

size_t packed_bytes(int M, int K) { return (size_t)((M + 15) / 16) * (K / 32) * 1024; }

__global__ __launch_bounds__(256) void pack_kernel(const uint16_t* __restrict__ W, int M, int K, int KC,
                                                   size_t total, uint4* __restrict__ out) {
  const size_t idx = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= total) return;
  const int lane = (int)(idx & 63);
  const size_t frag = idx >> 6;
  const int kc = (int)(frag % KC);
  const int rb = (int)(frag / KC);
  const int row = rb * 16 + (lane & 15);
  const int k = kc * 32 + 8 * (lane >> 4);
  uint4 v = make_uint4(0, 0, 0, 0);
  if (row < M) v = *(const uint4*)(W + (size_t)row * K + k);
  out[idx] = v;
}

hipError_t launch_pack_bf16(const uint16_t* W, int M, int K, void* out, hipStream_t s) {
  const int KC = K / 32;
  const size_t total = (size_t)((M + 15) / 16) * KC * 64;
  pack_kernel<<<(unsigned)((total + 255) / 256), 256, 0, s>>>(W, M, K, KC, total, (uint4*)out);
  return hipGetLastError();
}

// ------------------------------------------------------------------ GEMM, bf16 on matrix cores
//
// Y^T[o][n] = sum_k W[o][k] A[n][k] with v_mfma_f32_16x16x32_bf16: W fragment
// is the A operand (16 rows x 32 k), activations the B operand (32 k x 16
// nodes).  One workgroup owns a 16-row block and every node; its 4 waves take
// consecutive quarters of K and reduce through LDS in a fixed order, so every
// output is computed the same way whatever the node count or a node's slot.

template <int NT, int KIND>
__global__ __launch_bounds__(256) void gemm_mfma_kernel(const u32x4* __restrict__ Wp, int KC,
                                                        const uint16_t* __restrict__ act, int lda, size_t plane,
                                                        Epi ep) {
  __shared__ f32x4 red[4][NT][64];
  const int rb = blockIdx.x, w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int kc0 = (w * KC) >> 2, kc1 = ((w + 1) * KC) >> 2;
  f32x4 acc[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) acc[t] = (f32x4){0.f, 0.f, 0.f, 0.f};
  const u32x4* wp = Wp + (size_t)rb * KC * 64 + lane;
  const uint16_t* ap = act + (size_t)(lane & 15) * lda + 8 * (lane >> 4);
  constexpr int U = 8;
  int kc = kc0;
  for (; kc + U <= kc1; kc += U) {
    u32x4 wf[U];
#pragma unroll
    for (int u = 0; u < U; ++u) wf[u] = __builtin_nontemporal_load(wp + (size_t)(kc + u) * 64);
#pragma unroll
    for (int u = 0; u < U; ++u) {
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        const uint16_t* at = ap + (size_t)16 * t * lda + (kc + u) * 32;
        const u32x4 b = *(const u32x4*)at;
        const u32x4 bl = *(const u32x4*)(at + plane);
        acc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, wf[u]),
                                                         __builtin_bit_cast(bf16x8, b), acc[t], 0, 0, 0);
        acc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, wf[u]),
                                                         __builtin_bit_cast(bf16x8, bl), acc[t], 0, 0, 0);
      }
    }
  }
  for (; kc < kc1; ++kc) {
    const u32x4 wf = __builtin_nontemporal_load(wp + (size_t)kc * 64);
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      const uint16_t* at = ap + (size_t)16 * t * lda + kc * 32;
      const u32x4 b = *(const u32x4*)at;
      const u32x4 bl = *(const u32x4*)(at + plane);
      acc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, wf),
                                                       __builtin_bit_cast(bf16x8, b), acc[t], 0, 0, 0);
      acc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, wf),
                                                       __builtin_bit_cast(bf16x8, bl), acc[t], 0, 0, 0);
    }
  }
#pragma unroll
  for (int t = 0; t < NT; ++t) red[w][t][lane] = acc[t];
  __syncthreads();
  // D layout: lane l holds rows 4(l/16)+r, column (node) l%16
  const int l2 = threadIdx.x >> 2, r = threadIdx.x & 3;
  const int row = 4 * (l2 >> 4) + r, o = rb * 16 + row;
#pragma unroll
  for (int t = 0; t < NT; ++t) {
    const float s = ((red[0][t][l2][r] + red[1][t][l2][r]) + red[2][t][l2][r]) + red[3][t][l2][r];
    const int node = 16 * t + (l2 & 15);
    if (o < ep.M && node < ep.N) epilogue<uint16_t, KIND>(ep, node, o, s);
  }
}

template <int NT>
static void gemm_mfma_nt(int kind, const void* Wp, int M, int KC, const uint16_t* act, int lda, size_t plane,
                         const Epi& ep, hipStream_t s) {
  const int RB = (M + 15) / 16;
  const u32x4* w = (const u32x4*)Wp;
  switch (kind) {
    case EPI_QKV: gemm_mfma_kernel<NT, EPI_QKV><<<RB, 256, 0, s>>>(w, KC, act, lda, plane, ep); break;
    case EPI_RESID: gemm_mfma_kernel<NT, EPI_RESID><<<RB, 256, 0, s>>>(w, KC, act, lda, plane, ep); break;
    case EPI_GELU: gemm_mfma_kernel<NT, EPI_GELU><<<RB, 256, 0, s>>>(w, KC, act, lda, plane, ep); break;
    default: gemm_mfma_kernel<NT, EPI_LOGITS><<<RB, 256, 0, s>>>(w, KC, act, lda, plane, ep); break;
  }
}

hipError_t launch_gemm_mfma(int kind, const void* Wp, int M, int K, const uint16_t* act, int lda, size_t plane,
                            const Epi& ep, hipStream_t s) {
  const int KC = K / 32;
  if (ep.N <= 16) gemm_mfma_nt<1>(kind, Wp, M, KC, act, lda, plane, ep, s);
  else if (ep.N <= 32) gemm_mfma_nt<2>(kind, Wp, M, KC, act, lda, plane, ep, s);
  else if (ep.N <= 64) gemm_mfma_nt<4>(kind, Wp, M, KC, act, lda, plane, ep, s);
  else if (ep.N <= 128) gemm_mfma_nt<8>(kind, Wp, M, KC, act, lda, plane, ep, s);
  else if (ep.N <= 256) gemm_mfma_nt<16>(kind, Wp, M, KC, act, lda, plane, ep, s);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

// ------------------------------------------------------------------ GEMM, bf16 on the vector ALU
//
// Same packed fragments and work split as the matrix-core kernel; each lane
// multiplies its 8 weights into fp32 accumulators for every node, then the 4
// lanes sharing a row and the 4 waves are reduced in a fixed order.

template <int NV, int KIND>
__global__ __launch_bounds__(256) void gemm_vec_kernel(const u32x4* __restrict__ Wp, int KC,
                                                       const uint16_t* __restrict__ act, int lda, size_t plane,
                                                       Epi ep) {
  __shared__ float red[4][NV][16];
  const int rb = blockIdx.x, w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int kc0 = (w * KC) >> 2, kc1 = ((w + 1) * KC) >> 2;
  float acc[NV];
#pragma unroll
  for (int n = 0; n < NV; ++n) acc[n] = 0.f;
  const u32x4* wp = Wp + (size_t)rb * KC * 64 + lane;
  const uint16_t* ap = act + 8 * (lane >> 4);
  constexpr int U = 4;
  int kc = kc0;
  for (; kc < kc1; kc += U) {
    u32x4 wf[U];
#pragma unroll
    for (int u = 0; u < U; ++u)
      wf[u] = (kc + u < kc1) ? __builtin_nontemporal_load(wp + (size_t)(kc + u) * 64) : (u32x4){0, 0, 0, 0};
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (kc + u >= kc1) break;
      float wv[8];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        wv[2 * e] = __uint_as_float(wf[u][e] << 16);
        wv[2 * e + 1] = __uint_as_float(wf[u][e] & 0xffff0000u);
      }
#pragma unroll
      for (int n = 0; n < NV; ++n) {
        const uint16_t* an = ap + (size_t)n * lda + (kc + u) * 32;
        const u32x4 av = *(const u32x4*)an;
        const u32x4 al = *(const u32x4*)(an + plane);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float a0 = __uint_as_float(av[e] << 16) + __uint_as_float(al[e] << 16);
          const float a1 = __uint_as_float(av[e] & 0xffff0000u) + __uint_as_float(al[e] & 0xffff0000u);
          acc[n] = fmaf(wv[2 * e], a0, acc[n]);
          acc[n] = fmaf(wv[2 * e + 1], a1, acc[n]);
        }
      }
    }
  }
#pragma unroll
  for (int n = 0; n < NV; ++n) {
    acc[n] += __shfl_xor(acc[n], 16);
    acc[n] += __shfl_xor(acc[n], 32);
  }
  if (lane < 16) {
#pragma unroll
    for (int n = 0; n < NV; ++n) red[w][n][lane] = acc[n];
  }
  __syncthreads();
  for (int idx = threadIdx.x; idx < NV * 16; idx += 256) {
    const int n = idx >> 4, row = idx & 15, o = rb * 16 + row;
    const float s = ((red[0][n][row] + red[1][n][row]) + red[2][n][row]) + red[3][n][row];
    if (o < ep.M && n < ep.N) epilogue<uint16_t, KIND>(ep, n, o, s);
  }
}

template <int NV>
static void gemm_vec_nv(int kind, const void* Wp, int M, int KC, const uint16_t* act, int lda, size_t plane,
                        const Epi& ep, hipStream_t s) {
  const int RB = (M + 15) / 16;
  const u32x4* w = (const u32x4*)Wp;
  switch (kind) {
    case EPI_QKV: gemm_vec_kernel<NV, EPI_QKV><<<RB, 256, 0, s>>>(w, KC, act, lda, plane, ep); break;
    case EPI_RESID: gemm_vec_kernel<NV, EPI_RESID><<<RB, 256, 0, s>>>(w, KC, act, lda, plane, ep); break;
    case EPI_GELU: gemm_vec_kernel<NV, EPI_GELU><<<RB, 256, 0, s>>>(w, KC, act, lda, plane, ep); break;
    default: gemm_vec_kernel<NV, EPI_LOGITS><<<RB, 256, 0, s>>>(w, KC, act, lda, plane, ep); break;
  }
}

hipError_t launch_gemm_vec(int kind, const void* Wp, int M, int K, const uint16_t* act, int lda, size_t plane,
                           const Epi& ep, hipStream_t s) {
  const int KC = K / 32;
  if (ep.N <= 1) gemm_vec_nv<1>(kind, Wp, M, KC, act, lda, plane, ep, s);
  else if (ep.N <= 2) gemm_vec_nv<2>(kind, Wp, M, KC, act, lda, plane, ep, s);
  else if (ep.N <= 4) gemm_vec_nv<4>(kind, Wp, M, KC, act, lda, plane, ep, s);
  else if (ep.N <= 8) gemm_vec_nv<8>(kind, Wp, M, KC, act, lda, plane, ep, s);
  else if (ep.N <= 16) gemm_vec_nv<16>(kind, Wp, M, KC, act, lda, plane, ep, s);
  else return hipErrorInvalidValue;
  return hipGetLastError();
}

// ------------------------------------------------------------------ tree attention
//
// Keys of node i: cache rows 0..P-1, then its ancestors and itself in the tree
// scratch (ancestor bitmask).  Grid (head, split): splits 0..S-1 take 64
// cache rows each, splits S.. take 64 tree rows each.  A split loads its K/V
// tile into LDS once and scores it against every node; each (node, head,
// split) leaves a partial (max, sum of exp, unnormalised output) that the
// combine kernel merges in split order.  Split boundaries are absolute key
// positions, so a node's result does not depend on the node count.

template <typename T, int DH>
__global__ __launch_bounds__(256) void attn_partial_kernel(AttnArgs a) {
  __shared__ float Ks[64][DH + 1];
  __shared__ float Vs[64][DH + 1];
  __shared__ float es[4][64];
  const int h = blockIdx.x, s = blockIdx.y;
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const bool tree = s >= a.S;
  const int key0 = tree ? (s - a.S) * 64 : s * 64;
  const int nk = tree ? min(64, a.N - key0) : min(64, a.P - key0);
  const T* kb = tree ? (const T*)a.kt + ((size_t)h * a.max_nodes + key0) * DH
                     : (const T*)a.kc + ((size_t)h * a.max_ctx + key0) * DH;
  const T* vb = tree ? (const T*)a.vt + ((size_t)h * a.max_nodes + key0) * DH
                     : (const T*)a.vc + ((size_t)h * a.max_ctx + key0) * DH;
  for (int idx = threadIdx.x; idx < 64 * DH; idx += 256) {
    const int j = idx / DH, c = idx - j * DH;
    float kv = 0.f, vv = 0.f;
    if (j < nk) {
      kv = ldT(kb, (size_t)j * DH + c);
      vv = ldT(vb, (size_t)j * DH + c);
    }
    Ks[j][c] = kv;
    Vs[j][c] = vv;
  }
  __syncthreads();
  for (int n0 = 0; n0 < a.N; n0 += 4) {
    const int n = n0 + w;
    if (n < a.N) {
      const float* qn = a.q + (size_t)n * a.d + h * DH;
      bool valid = lane < nk;
      if (tree && valid) {
        const int j = key0 + lane;
        valid = (a.anc[(size_t)n * a.W + (j >> 6)] >> (j & 63)) & 1ull;
      }
      float dot = 0.f;
#pragma unroll 8
      for (int c = 0; c < DH; ++c) dot = fmaf(qn[c], Ks[lane][c], dot);
      const float sc = valid ? dot * a.scale : -INFINITY;
      const float m = wave_max(sc);
      float* out = a.part + (((size_t)h * a.NS + s) * a.N + n) * (DH + 2);
      if (m == -INFINITY) {
        if (lane < DH) out[2 + lane] = 0.f;
        if (lane == 0) {
          out[0] = -INFINITY;
          out[1] = 0.f;
        }
      } else {
        const float e = valid ? expf(sc - m) : 0.f;
        const float z = wave_sum(e);
        es[w][lane] = e;
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
        if (lane < DH) {
          float o = 0.f;
#pragma unroll 8
          for (int j = 0; j < 64; ++j) o = fmaf(es[w][j], Vs[j][lane], o);
          out[2 + lane] = o;
        }
        if (lane == 0) {
          out[0] = m;
          out[1] = z;
        }
      }
    }
    __syncthreads();
  }
}

template <int DH, typename OUT>
__global__ __launch_bounds__(256) void attn_combine_kernel(const float* __restrict__ part, int NS, int N, int H,
                                                           int d, OUT* __restrict__ out, int ldo, size_t plane) {
  const int pair = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (pair >= N * H) return;
  const int n = pair / H, h = pair - n * H;
  const size_t stride = (size_t)N * (DH + 2);
  const float* p = part + ((size_t)h * NS * N + n) * (DH + 2);
  float m = -INFINITY;
  for (int s = 0; s < NS; ++s) m = fmaxf(m, p[s * stride]);
  float z = 0.f, o = 0.f;
  for (int s = 0; s < NS; ++s) {
    const float ms = p[s * stride];
    if (ms == -INFINITY) continue;
    const float wgt = expf(ms - m);
    z = fmaf(p[s * stride + 1], wgt, z);
    if (lane < DH) o = fmaf(p[s * stride + 2 + lane], wgt, o);
  }
  if (lane < DH) st_act(out, (size_t)n * ldo + h * DH + lane, plane, o / z);
}

hipError_t launch_attn(int f32, int DH, const AttnArgs& a, hipStream_t s) {
  dim3 grid(a.H, a.NS);
  if (f32) {
    if (DH == 64) attn_partial_kernel<float, 64><<<grid, 256, 0, s>>>(a);
    else attn_partial_kernel<float, 32><<<grid, 256, 0, s>>>(a);
  } else {
    if (DH == 64) attn_partial_kernel<uint16_t, 64><<<grid, 256, 0, s>>>(a);
    else attn_partial_kernel<uint16_t, 32><<<grid, 256, 0, s>>>(a);
  }
  return hipGetLastError();
}

hipError_t launch_attn_combine(int f32, int DH, const float* part, int NS, int N, int H, int d, void* out, int ldo,
                               size_t plane, hipStream_t s) {
  const int blocks = (N * H + 3) / 4;
  if (f32) {
    if (DH == 64) attn_combine_kernel<64, float><<<blocks, 256, 0, s>>>(part, NS, N, H, d, (float*)out, ldo, 0);
    else attn_combine_kernel<32, float><<<blocks, 256, 0, s>>>(part, NS, N, H, d, (float*)out, ldo, 0);
  } else {
    if (DH == 64)
      attn_combine_kernel<64, uint16_t><<<blocks, 256, 0, s>>>(part, NS, N, H, d, (uint16_t*)out, ldo, plane);
    else
      attn_combine_kernel<32, uint16_t><<<blocks, 256, 0, s>>>(part, NS, N, H, d, (uint16_t*)out, ldo, plane);
  }
  return hipGetLastError();
}

// ------------------------------------------------------------------ accept: greedy

// argmax of each logits row, lowest index among equal maxima
__global__ __launch_bounds__(256) void argmax_kernel(const float* __restrict__ logits, int V, int* __restrict__ g) {
  __shared__ float sv[256];
  __shared__ int si[256];
  const int n = blockIdx.x;
  const float* row = logits + (size_t)n * V;
  float best = -INFINITY;
  int bi = V;
  for (int v = threadIdx.x; v < V; v += 256) {
    const float x = row[v];
    if (x > best || (x == best && v < bi)) {
      best = x;
      bi = v;
    }
  }
  sv[threadIdx.x] = best;
  si[threadIdx.x] = bi;
  __syncthreads();
  for (int off = 128; off > 0; off >>= 1) {
    if (threadIdx.x < off) {
      const float ov = sv[threadIdx.x + off];
      const int oi = si[threadIdx.x + off];
      if (ov > sv[threadIdx.x] || (ov == sv[threadIdx.x] && oi < si[threadIdx.x])) {
        sv[threadIdx.x] = ov;
        si[threadIdx.x] = oi;
      }
    }
    __syncthreads();
  }
  if (threadIdx.x == 0) g[n] = si[0] < V ? si[0] : 0;
}

// one thread: matched = parent matched and token == parent's argmax; keep the
// deepest matched node (lowest index among equals)
__global__ void greedy_walk_kernel(const int* __restrict__ tokens, const int* __restrict__ parents,
                                   const int* __restrict__ depth, int N, const int* __restrict__ g,
                                   int* __restrict__ path, int* __restrict__ path_len, int* __restrict__ next) {
  __shared__ unsigned char m[1024];
  if (threadIdx.x != 0) return;
  m[0] = 1;
  int best = 0;
  for (int i = 1; i < N; ++i) {
    const int p = parents[i];
    m[i] = m[p] && tokens[i] == g[p];
    if (m[i] && depth[i] > depth[best]) best = i;
  }
  const int len = depth[best] + 1;
  int j = best;
  for (int t = len - 1; t >= 0; --t) {
    path[t] = j;
    j = parents[j];
  }
  *path_len = len;
  *next = g[best];
}

hipError_t launch_argmax(const float* logits, int N, int V, int* g, hipStream_t s) {
  argmax_kernel<<<N, 256, 0, s>>>(logits, V, g);
  return hipGetLastError();
}

hipError_t launch_greedy_walk(const int* tokens, const int* parents, const int* depth, int N, const int* g,
                              int* path, int* path_len, int* next, hipStream_t s) {
  greedy_walk_kernel<<<1, 64, 0, s>>>(tokens, parents, depth, N, g, path, path_len, next);
  return hipGetLastError();
}

// ------------------------------------------------------------------ accept: rejection sampling
//
// Philox4x64-10 (Salmon, Moraes, Dror, Shaw, SC'11): 10 rounds of two 64x64
// multiplies with the published multipliers, key bumped by the published Weyl
// constants between rounds.

__device__ double philox_uniform(uint64_t seed, uint64_t stream, uint64_t ctr0) {
  const uint64_t M0 = 0xD2E7470EE14C6C93ull, M1 = 0xCA5A826395121157ull;
  const uint64_t W0 = 0x9E3779B97F4A7C15ull, W1 = 0xBB67AE8584CAA73Bull;
  uint64_t c0 = ctr0, c1 = 0, c2 = 0, c3 = 0, k0 = seed, k1 = stream;
  for (int r = 0; r < 10; ++r) {
    if (r) {
      k0 += W0;
      k1 += W1;
    }
    const uint64_t h0 = __umul64hi(M0, c0), l0 = M0 * c0;
    const uint64_t h1 = __umul64hi(M1, c2), l1 = M1 * c2;
    const uint64_t n0 = h1 ^ c1 ^ k0, n2 = h0 ^ c3 ^ k1;
    c0 = n0;
    c1 = l1;
    c2 = n2;
    c3 = l0;
  }
  return (double)(c0 >> 11) * 0x1.0p-53;
}

#define SA_THREADS 1024

// every thread sums its contiguous chunk of the vocabulary in index order;
// chunk sums are then added pairwise in a fixed tree
__device__ double block_sum_chunks(double v, double* red) {
  red[threadIdx.x] = v;
  __syncthreads();
  for (int off = SA_THREADS / 2; off > 0; off >>= 1) {
    if (threadIdx.x < off) red[threadIdx.x] = red[threadIdx.x] + red[threadIdx.x + off];
    __syncthreads();
  }
  const double r = red[0];
  __syncthreads();
  return r;
}

__device__ double block_max_d(double v, double* red) {
  red[threadIdx.x] = v;
  __syncthreads();
  for (int off = SA_THREADS / 2; off > 0; off >>= 1) {
    if (threadIdx.x < off) red[threadIdx.x] = fmax(red[threadIdx.x], red[threadIdx.x + off]);
    __syncthreads();
  }
  const double r = red[0];
  __syncthreads();
  return r;
}

__global__ __launch_bounds__(SA_THREADS) void sample_accept_kernel(
    const int* __restrict__ tokens, const int* __restrict__ parents, int N, int V, const float* __restrict__ logits,
    const float* __restrict__ draft, double T, uint64_t seed, int wor, double* __restrict__ r, double* __restrict__ p,
    double* __restrict__ qq, int* __restrict__ path, int* __restrict__ path_len, int* __restrict__ next) {
  __shared__ double red[SA_THREADS];
  __shared__ int sh_choice;
  const int tid = threadIdx.x;
  const int C = (V + SA_THREADS - 1) / SA_THREADS;
  const int v0 = tid * C, v1 = min(V, v0 + C);
  int u = 0, len = 1;
  if (tid == 0) path[0] = 0;
  double Z = 1.0;
  for (;;) {
    const float* row = logits + (size_t)u * V;
    double mx = -INFINITY;
    for (int v = v0; v < v1; ++v) mx = fmax(mx, (double)row[v] / T);
    mx = block_max_d(mx, red);
    double s = 0.0;
    for (int v = v0; v < v1; ++v) {
      const double e = exp((double)row[v] / T - mx);
      p[v] = e;
      s += e;
    }
    const double S = block_sum_chunks(s, red);
    const float* q = draft + (size_t)u * V;
    double sq = 0.0;
    for (int v = v0; v < v1; ++v) {
      p[v] = p[v] / S;
      r[v] = p[v];
      qq[v] = (double)q[v];
      sq += qq[v];
    }
    double Zq = block_sum_chunks(sq, red);  // includes the barrier that publishes r, qq
    Z = 1.0;
    int accepted = -1;
    for (int c = u + 1; c < N; ++c) {
      if (parents[c] != u) continue;
      const int x = tokens[c];
      const double U = philox_uniform(seed, 0, (uint64_t)c);
      const double rx = r[x], qx = qq[x];
      const bool acc = (qx == 0.0) ? (rx > 0.0) : (U < (rx / Z) / (qx / Zq));
      if (acc) {
        accepted = c;
        break;
      }
      __syncthreads();  // everyone has read r[x], qq[x]
      double nz = 0.0;
      for (int v = v0; v < v1; ++v) {
        const double t = r[v] / Z - qq[v] / Zq;
        r[v] = t > 0.0 ? t : 0.0;
        nz += r[v];
      }
      Z = block_sum_chunks(nz, red);
      if (wor) {
        if (tid == 0) qq[x] = 0.0;
        __syncthreads();
        double s2 = 0.0;
        for (int v = v0; v < v1; ++v) s2 += qq[v];
        Zq = block_sum_chunks(s2, red);
      }
    }
    if (accepted < 0) break;
    if (tid == 0) path[len] = accepted;
    ++len;
    u = accepted;
    __syncthreads();
  }
  // extra token: smallest v whose running sum exceeds U * Z
  const double U2 = philox_uniform(seed, 1, (uint64_t)u);
  const bool use_r = Z > 0.0;
  const double* w = use_r ? r : p;
  const double target = U2 * (use_r ? Z : 1.0);
  double cs = 0.0;
  int lastpos = -1;
  for (int v = v0; v < v1; ++v) {
    cs += w[v];
    if (w[v] > 0.0) lastpos = v;
  }
  red[tid] = cs;
  __shared__ int last_sh[SA_THREADS];
  last_sh[tid] = lastpos;
  __syncthreads();
  if (tid == 0) {
    double run = 0.0;
    int choice = -1, last = 0;
    for (int t = 0; t < SA_THREADS && choice < 0; ++t) {
      if (last_sh[t] >= 0) last = last_sh[t];
      if (run + red[t] > target) {
        const int a = t * C, b = min(V, a + C);
        double c2 = run;
        for (int v = a; v < b; ++v) {
          c2 += w[v];
          if (c2 > target) {
            choice = v;
            break;
          }
        }
      }
      run += red[t];
    }
    if (choice < 0) {
      for (int t = SA_THREADS - 1; t >= 0; --t)
        if (last_sh[t] >= 0) {
          last = last_sh[t];
          break;
        }
      choice = last;
    }
    sh_choice = choice;
    *path_len = len;
    *next = choice;
  }
}

hipError_t launch_sample_accept(const int* tokens, const int* parents, int N, int V, const float* logits,
                                const float* draft, double temperature, uint64_t seed, int wor, double* r, double* p,
                                double* qq, int* path, int* path_len, int* next, hipStream_t s) {
  sample_accept_kernel<<<1, SA_THREADS, 0, s>>>(tokens, parents, N, V, logits, draft, temperature, seed, wor, r, p,
                                                qq, path, path_len, next);
  return hipGetLastError();
}

// ------------------------------------------------------------------ KV commit

template <typename T>
__global__ __launch_bounds__(256) void commit_kernel(T* __restrict__ kc, T* __restrict__ vc,
                                                     const T* __restrict__ kt, const T* __restrict__ vt, int max_ctx,
                                                     int max_nodes, int DH, int P, const int* __restrict__ path,
                                                     const int* __restrict__ path_len, unsigned* __restrict__ err) {
  const int lh = blockIdx.x;
  const int len = *path_len;
  if (len < 0 || len > max_nodes) {
    if (lh == 0 && threadIdx.x == 0) atomicAdd(err, 1u);
    return;
  }
  for (int idx = threadIdx.x; idx < len * DH; idx += 256) {
    const int t = idx / DH, c = idx - t * DH;
    const int node = path[t];
    if (node < 0 || node >= max_nodes || P + t >= max_ctx) {
      if (c == 0 && lh == 0) atomicAdd(err, 1u);
      continue;
    }
    const size_t dst = ((size_t)lh * max_ctx + P + t) * DH + c;
    const size_t src = ((size_t)lh * max_nodes + node) * DH + c;
    kc[dst] = kt[src];
    vc[dst] = vt[src];
  }
}

hipError_t launch_commit(int f32, void* kc, void* vc, const void* kt, const void* vt, int LH, int max_ctx,
                         int max_nodes, int DH, int P, const int* path, const int* path_len, unsigned* err,
                         hipStream_t s) {
  if (f32)
    commit_kernel<float><<<LH, 256, 0, s>>>((float*)kc, (float*)vc, (const float*)kt, (const float*)vt, max_ctx,
                                            max_nodes, DH, P, path, path_len, err);
  else
    commit_kernel<uint16_t><<<LH, 256, 0, s>>>((uint16_t*)kc, (uint16_t*)vc, (const uint16_t*)kt,
                                               (const uint16_t*)vt, max_ctx, max_nodes, DH, P, path, path_len, err);
  return hipGetLastError();
}

}  // namespace ssd
