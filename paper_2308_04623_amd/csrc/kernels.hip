// HIP kernels of libssd for CDNA4 (gfx950): one decoder pass over a token
// tree (Sec. 3.1 of Spector & Re, arXiv 2308.04623), the accept/reject walk
// (Sec. 2.3) and the KV commit.
//
// Data layout (HBM):
//   x        fp32 [N][d]         residual stream
//   q        fp32 [N][d]         queries of the current layer
//   act_*    GEMM inputs [Npad][d or d_mlp]: fp32 rows for fp32 models; float16
//            in matrix-core fragment order for bf16 models (see st_act)
//   part     fp32 [S][N][d]      split-K partial sums of the residual GEMMs
//   K/V      storage type [L][H][rows][DH] (cache rows: positions; scratch rows: nodes)
//   packed W 16x32 float16 fragments (the bf16 weights converted: exact for 0
//            and magnitudes in [2^-17, 65504], within 2^-25 below);
//            fragment (rb, kc) holds rows 16rb.., k 32kc..,
//            lane l's 16 bytes = W[16rb + l%16][32kc + 8(l/16) .. +8], fragments
//            ordered rb-major so one wave streams 1 KB contiguous per load.
//            8-bit models: the same fragments at half size (512 B), lane l's
//            8 bytes = the codes of the same 8 weights plus 128, and a float32
//            scale per row; the weight is scale * code.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include <type_traits>

#include "ssd_internal.h"

namespace ssd {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef float f32x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned u32x2 __attribute__((ext_vector_type(2)));

// ------------------------------------------------------------------ helpers

__device__ __forceinline__ float bf2f(uint16_t h) { return __uint_as_float((uint32_t)h << 16); }

// float -> bfloat16, round to nearest even (v_cvt_pk_bf16_f32)
__device__ __forceinline__ uint16_t f2bf(float f) { return __builtin_bit_cast(uint16_t, (__bf16)f); }
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef unsigned u32x2 __attribute__((ext_vector_type(2)));
// two floats -> packed bfloat16 pair (first in the low half), one instruction
__device__ __forceinline__ uint32_t f2bf2(float a, float b) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t){a, b}, bf16x2_t));
}

template <typename T> __device__ __forceinline__ float ldT(const T* p, size_t i);
template <> __device__ __forceinline__ float ldT<float>(const float* p, size_t i) { return p[i]; }
template <> __device__ __forceinline__ float ldT<uint16_t>(const uint16_t* p, size_t i) { return bf2f(p[i]); }

template <typename T> __device__ __forceinline__ void stT(T* p, size_t i, float v);
template <typename T, int E> __device__ __forceinline__ float ldT(const T (&r)[E], int i) { return ldT((const T*)r, (size_t)i); }
template <> __device__ __forceinline__ void stT<float>(float* p, size_t i, float v) { p[i] = v; }
template <> __device__ __forceinline__ void stT<uint16_t>(uint16_t* p, size_t i, float v) { p[i] = f2bf(v); }

// GEMM inputs.  fp32 models: plain rows, element (n, k) at n * ld + k.
// bf16 models: float16 (11 significant bits, round to nearest even) in
// matrix-core fragment order, so that one wave's load of a 16-node x 32-k
// operand fragment is 1 KB contiguous: element (n, k) lives in fragment
// f = (n/16) * ld + k/32 (ld = K/32), lane (n%16) + 16 ((k%32)/8), position
// k%8.  The weights are multiplied as float16 too: their packed copies are
// the bf16 values converted to float16 (exact for 0 and magnitudes in
// [2^-17, 65504]; see pack_kernel).
// A float16 operand past the type's range (|v| > 65504, or NaN) would enter
// the matrix cores as inf or NaN: such an element is counted in err (the
// session's error counter) and stored as converted.
template <typename T> __device__ __forceinline__ void st_act(T* p, int n, int k, int ld, float v, unsigned* err);
template <> __device__ __forceinline__ void st_act<float>(float* p, int n, int k, int ld, float v, unsigned*) {
  p[(size_t)n * ld + k] = v;
}
template <>
__device__ __forceinline__ void st_act<uint16_t>(uint16_t* p, int n, int k, int ld, float v, unsigned* err) {
  const size_t f = (size_t)(n >> 4) * ld + (k >> 5);
  // (one count per wave and call: the lowest lane out of range adds 1)
  const unsigned long long m = __builtin_amdgcn_ballot_w64(!(fabsf(v) <= 65504.f));
  if (m && err && (int)__builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, 0u)) == __builtin_ctzll(m)) atomicAdd(err, 1u);
  p[f * 512 + ((n & 15) + 16 * ((k & 31) >> 3)) * 8 + (k & 7)] = __builtin_bit_cast(uint16_t, (_Float16)v);
}
__device__ __forceinline__ float h2f(uint16_t h) { return (float)__builtin_bit_cast(_Float16, h); }
// four consecutive columns k .. k + 3 (k a multiple of 4) of row n in the
// GEMM-input layout: one 8-byte store, out-of-range values counted as st_act does
__device__ __forceinline__ void st_act4_u16(uint16_t* p, int n, int k, int ld, const float (&v)[4], unsigned* err) {
  const size_t f = (size_t)(n >> 4) * ld + (k >> 5);
  const bool bad = !(fabsf(v[0]) <= 65504.f) || !(fabsf(v[1]) <= 65504.f) || !(fabsf(v[2]) <= 65504.f) ||
                   !(fabsf(v[3]) <= 65504.f);
  const unsigned long long m = __builtin_amdgcn_ballot_w64(bad);
  if (m && err && (int)__builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, 0u)) == __builtin_ctzll(m)) atomicAdd(err, 1u);
  const uint32_t lo = (uint32_t)__builtin_bit_cast(uint16_t, (_Float16)v[0]) |
                      ((uint32_t)__builtin_bit_cast(uint16_t, (_Float16)v[1]) << 16);
  const uint32_t hi = (uint32_t)__builtin_bit_cast(uint16_t, (_Float16)v[2]) |
                      ((uint32_t)__builtin_bit_cast(uint16_t, (_Float16)v[3]) << 16);
  *(u32x2*)(p + f * 512 + ((n & 15) + 16 * ((k & 31) >> 3)) * 8 + (k & 7)) = (u32x2){lo, hi};
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

// ------------------------------------------------------------------ pass signals

__device__ __forceinline__ unsigned xcc_id() {
  unsigned x;
  asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(x));
  return x & 15;
}

// one relaxed device-scope increment by thread 0 of block (0, 0)
__device__ __forceinline__ void pass_signal(unsigned long long* sig) {
  if (sig && blockIdx.x == 0 && blockIdx.y == 0 && threadIdx.x == 0)
    __hip_atomic_fetch_add(sig, 1ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
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
                                                    int d, float* __restrict__ x, unsigned long long* sig,
                                                    unsigned* xcc0) {
  if (sig && blockIdx.x == 0 && threadIdx.x == 0) {
    // the XCD of block 0, stored before the first signal of the pass is released
    __hip_atomic_store(xcc0, xcc_id(), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __hip_atomic_fetch_add(sig, 1ull, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_AGENT);
  }
  const int n = blockIdx.x;
  const size_t t = (size_t)tokens[n] * d, p = (size_t)pos[n] * d;
  for (int k = threadIdx.x; k < d; k += blockDim.x) x[(size_t)n * d + k] = ldT(wte, t + k) + ldT(wpe, p + k);
}

hipError_t launch_embed(int f32, const void* wte, const void* wpe, const int* tokens, const int* pos, int N, int d,
                        float* x, unsigned long long* sig, unsigned* xcc0, hipStream_t s) {
  if (sig && !xcc0) return hipErrorInvalidValue;
  if (f32)
    embed_kernel<float><<<N, 256, 0, s>>>((const float*)wte, (const float*)wpe, tokens, pos, d, x, sig, xcc0);
  else
    embed_kernel<uint16_t><<<N, 256, 0, s>>>((const uint16_t*)wte, (const uint16_t*)wpe, tokens, pos, d, x, sig,
                                             xcc0);
  return hipGetLastError();
}

// ------------------------------------------------------------------ residual + LayerNorm
//
// One workgroup per node, the row held in registers: thread t owns the
// column groups 4t .. 4t+3, 4(t+256) .. 4(t+256)+3, ... (E groups, E =
// ceil(d / 1024); d is a multiple of 32), so every load is 8 or 16 bytes and a
// bf16 model's activation store is one 8-byte write:
//   if S > 0:  x[n] += bias + part[0][n] + ... + part[S-1][n]   (split-K sums of the
//              previous residual GEMM, added in split order), written back;
//   a[n] = (x[n] - mean) / sqrt(var + eps) * g + b   (biased variance).
// Every load is issued (clamped to the row) before any of them is used, so
// the row costs one memory round trip.  SPL is the split count when known at
// compile time (0, 1, 2, 4 or 8), else -1 and the loop runs to S.

template <typename T> __device__ __forceinline__ void ld4(const T* p, size_t k, float (&o)[4]);
template <> __device__ __forceinline__ void ld4<float>(const float* p, size_t k, float (&o)[4]) {
  const f32x4 v = *(const f32x4*)(p + k);
  o[0] = v.x; o[1] = v.y; o[2] = v.z; o[3] = v.w;
}
template <> __device__ __forceinline__ void ld4<uint16_t>(const uint16_t* p, size_t k, float (&o)[4]) {
  const u32x2 v = *(const u32x2*)(p + k);
  o[0] = __uint_as_float(v.x << 16); o[1] = __uint_as_float(v.x & 0xffff0000u);
  o[2] = __uint_as_float(v.y << 16); o[3] = __uint_as_float(v.y & 0xffff0000u);
}
template <typename T> __device__ __forceinline__ void st_act4(T* p, int n, int k, int ld, const float (&v)[4], unsigned* err);
template <> __device__ __forceinline__ void st_act4<float>(float* p, int n, int k, int ld, const float (&v)[4], unsigned*) {
  *(f32x4*)(p + (size_t)n * ld + k) = (f32x4){v[0], v[1], v[2], v[3]};
}
template <>
__device__ __forceinline__ void st_act4<uint16_t>(uint16_t* p, int n, int k, int ld, const float (&v)[4], unsigned* err) {
  st_act4_u16(p, n, k, ld, v, err);
}

template <typename T, typename OUT, int E, int SPL>
__global__ __launch_bounds__(256) void ln_resid_kernel(float* __restrict__ x, int d, const float* __restrict__ part,
                                                       int S, size_t pstride, const T* __restrict__ bias,
                                                       const T* __restrict__ g, const T* __restrict__ b, float eps,
                                                       OUT* __restrict__ a, int lda, unsigned long long* sig,
                                                       unsigned* err) {
  constexpr int PS = SPL > 0 ? SPL : 1;
  __shared__ float red[4];
  pass_signal(sig);
  const int n = blockIdx.x, tid = threadIdx.x, nc = d >> 2;
  float* xr = x + (size_t)n * d;
  const float* pr = part + (size_t)n * d;
  float v[E][4], gw[E][4], bw[E][4], cw[E][4];
  float pv[E][PS][4];
#pragma unroll
  for (int i = 0; i < E; ++i) {
    const size_t k = 4 * (size_t)min(tid + i * 256, nc - 1);
    ld4(xr, k, v[i]);
    ld4(g, k, gw[i]);
    ld4(b, k, bw[i]);
    if constexpr (SPL > 0) {
      ld4(bias, k, cw[i]);
#pragma unroll
      for (int sp = 0; sp < SPL; ++sp) ld4(pr + sp * pstride, k, pv[i][sp]);
    }
  }
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < E; ++i) {
    const int c = tid + i * 256;
    if constexpr (SPL != 0) {
      float acc[4];
      if constexpr (SPL > 0) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          acc[j] = cw[i][j];
#pragma unroll
          for (int sp = 0; sp < SPL; ++sp) acc[j] += pv[i][sp][j];
        }
      } else {
        const size_t k = 4 * (size_t)min(c, nc - 1);
        ld4(bias, k, acc);
        for (int sp = 0; sp < S; ++sp) {
          float p4[4];
          ld4(pr + sp * pstride, k, p4);
#pragma unroll
          for (int j = 0; j < 4; ++j) acc[j] += p4[j];
        }
      }
#pragma unroll
      for (int j = 0; j < 4; ++j) v[i][j] += acc[j];
      if (c < nc) *(f32x4*)(xr + 4 * c) = (f32x4){v[i][0], v[i][1], v[i][2], v[i][3]};
    }
    if (c < nc) s += (v[i][0] + v[i][1]) + (v[i][2] + v[i][3]);
  }
  const float mean = block_sum256(s, red) / d;
  float q = 0.f;
#pragma unroll
  for (int i = 0; i < E; ++i)
    if (tid + i * 256 < nc) {
#pragma unroll
      for (int j = 0; j < 4; ++j) q += (v[i][j] - mean) * (v[i][j] - mean);
    }
  const float den = sqrtf(block_sum256(q, red) / d + eps);
#pragma unroll
  for (int i = 0; i < E; ++i) {
    const int c = tid + i * 256;
    float o[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) o[j] = (v[i][j] - mean) / den * gw[i][j] + bw[i][j];
    // (the bf16 store's error ballot runs over the in-range lanes only)
    if (c < nc) st_act4(a, n, 4 * c, lda, o, err);
  }
}

template <typename T, int E, int SPL>
static void ln_go(float* x, int N, int d, const float* part, int S, size_t pstride, const void* bias, const void* g,
                  const void* b, float eps, void* a, int lda, unsigned long long* sig, unsigned* err, hipStream_t s) {
  ln_resid_kernel<T, T, E, SPL><<<N, 256, 0, s>>>(x, d, part, S, pstride, (const T*)bias, (const T*)g, (const T*)b,
                                                  eps, (T*)a, lda, sig, err);
}

template <typename T, int E>
static void ln_go_s(float* x, int N, int d, const float* part, int S, size_t pstride, const void* bias,
                    const void* g, const void* b, float eps, void* a, int lda, unsigned long long* sig,
                    unsigned* err, hipStream_t s) {
  if (S == 0) ln_go<T, E, 0>(x, N, d, part, S, pstride, bias, g, b, eps, a, lda, sig, err, s);
  else if (S == 1) ln_go<T, E, 1>(x, N, d, part, S, pstride, bias, g, b, eps, a, lda, sig, err, s);
  else if (S == 2) ln_go<T, E, 2>(x, N, d, part, S, pstride, bias, g, b, eps, a, lda, sig, err, s);
  else if (S == 4) ln_go<T, E, 4>(x, N, d, part, S, pstride, bias, g, b, eps, a, lda, sig, err, s);
  else if (S == 8) ln_go<T, E, 8>(x, N, d, part, S, pstride, bias, g, b, eps, a, lda, sig, err, s);
  else ln_go<T, E, -1>(x, N, d, part, S, pstride, bias, g, b, eps, a, lda, sig, err, s);
}

template <typename T>
static hipError_t ln_go_e(float* x, int N, int d, const float* part, int S, size_t pstride, const void* bias,
                          const void* g, const void* b, float eps, void* a, int lda, unsigned long long* sig,
                          unsigned* err, hipStream_t s) {
  if (d % 32) return hipErrorInvalidValue;
  switch ((d + 1023) / 1024) {
    case 1: ln_go_s<T, 1>(x, N, d, part, S, pstride, bias, g, b, eps, a, lda, sig, err, s); break;
    case 2: ln_go_s<T, 2>(x, N, d, part, S, pstride, bias, g, b, eps, a, lda, sig, err, s); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_ln(int f32, float* x, int N, int d, const float* part, int S, size_t pstride, const void* bias,
                     const void* g, const void* b, float eps, void* a, int lda, unsigned long long* sig,
                     unsigned* err, hipStream_t s) {
  if (S > 0 && !bias) return hipErrorInvalidValue;
  if (f32) return ln_go_e<float>(x, N, d, part, S, pstride, bias, g, b, eps, a, lda, sig, err, s);
  return ln_go_e<uint16_t>(x, N, d, part, S, pstride, bias, g, b, eps, a, lda, sig, err, s);
}

// ------------------------------------------------------------------ GEMM epilogues

template <typename T, int KIND>
__device__ __forceinline__ void epilogue(const Epi& e, int n, int o, float acc) {
  const int nn = e.node0 + n;
  if (KIND == EPI_PARTIAL) {
    e.part[(size_t)e.split * e.part_stride + (size_t)nn * e.d + o] = acc;
    return;
  }
  const float y = acc + (e.bias ? ldT((const T*)e.bias, o) : 0.f);
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
    st_act((T*)e.out, nn, o, e.ldo, gelu_tanh(y), e.err);
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
                                                   size_t total, uint4* __restrict__ out, unsigned* __restrict__ bad) {
  const size_t idx = (size_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= total) return;
  const int lane = (int)(idx & 63);
  const size_t frag = idx >> 6;
  const int kc = (int)(frag % KC);
  const int rb = (int)(frag / KC);
  const int row = rb * 16 + (lane & 15);
  const int k = kc * 32 + 8 * (lane >> 4);
  u32x4 v = (u32x4){0, 0, 0, 0};
  if (row < M) v = *(const u32x4*)(W + (size_t)row * K + k);
  // bf16 -> float16, round to nearest even.  bf16 keeps 8 significant bits:
  // the conversion is exact for 0 and every magnitude in [2^-17, 65504]
  // (float16's subnormal spacing is 2^-24, so 8 significant bits need
  // |w| >= 2^-17); below 2^-17 the error is at most 2^-25 per weight.
  // Magnitudes past 65504 (or NaN) cannot be represented: they are counted
  // in bad and the model is refused.
  const f32x8 f = __builtin_convertvector(__builtin_bit_cast(bf16x8, v), f32x8);
  bool over = false;
#pragma unroll
  for (int e = 0; e < 8; ++e) over |= !(fabsf(f[e]) <= 65504.f);
  if (over) atomicAdd(bad, 1u);
  out[idx] = __builtin_bit_cast(uint4, __builtin_convertvector(f, f16x8));
}

hipError_t launch_pack_bf16(const uint16_t* W, int M, int K, void* out, unsigned* bad, hipStream_t s) {
  const int KC = K / 32;
  const size_t total = (size_t)((M + 15) / 16) * KC * 64;
  pack_kernel<<<(unsigned)((total + 255) / 256), 256, 0, s>>>(W, M, K, KC, total, (uint4*)out, bad);
  return hipGetLastError();
}

// 8-bit weights (symmetric, one float32 scale per row).  Per row, with a the
// largest magnitude (exact in float32), the codes are decided in float32,
// every operation rounded once to nearest even: r = 127 / a,
// code = clamp(rint(w r), -127, 127), scale = a / 127; a row with
// a < 2^-100 gets scale 0 and codes 0.  One workgroup per 16-row block: 16
// threads per row find a, then every thread writes 8-byte lane slots of the
// block's fragments (codes stored plus 128).  Rows past M get scale 0 and
// code 0; NaN or infinite weights are counted in bad.
__global__ __launch_bounds__(256) void pack_q8_kernel(const uint16_t* __restrict__ W, int M, int K, int KC,
                                                      u32x2* __restrict__ out, float* __restrict__ scales,
                                                      unsigned* __restrict__ bad) {
  __shared__ float rr[16];
  const int rb = blockIdx.x, tid = threadIdx.x, rl = tid >> 4, sub = tid & 15, row = rb * 16 + rl;
  float a = 0.f;
  int nf = 0;
  if (row < M)
    for (int k = sub; k < K; k += 16) {
      const float v = bf2f(W[(size_t)row * K + k]);
      nf |= !isfinite(v);
      a = fmaxf(a, fabsf(v));
    }
#pragma unroll
  for (int m = 1; m < 16; m <<= 1) {
    a = fmaxf(a, __shfl_xor(a, m));
    nf |= __shfl_xor(nf, m);
  }
  if (sub == 0) {
    if (nf) atomicAdd(bad, 1u);
    const bool live = row < M && a >= 0x1p-100f;
    rr[rl] = live ? 127.0f / a : 0.f;
    scales[row] = live ? a / 127.0f : 0.f;
  }
  __syncthreads();
  for (int idx = tid; idx < KC * 64; idx += 256) {
    const int kc = idx >> 6, lane = idx & 63, r = lane & 15, k = kc * 32 + 8 * (lane >> 4);
    u32x2 b = (u32x2){0x80808080u, 0x80808080u};
    if (rb * 16 + r < M) {
      const u32x4 v = *(const u32x4*)(W + (size_t)(rb * 16 + r) * K + k);
      const f32x8 f = __builtin_convertvector(__builtin_bit_cast(bf16x8, v), f32x8);
      const float rv = rr[r];
      b = (u32x2){0u, 0u};
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float c = fminf(fmaxf(rintf(f[e] * rv), -127.f), 127.f);
        b[e >> 2] |= (unsigned)((int)c + 128) << (8 * (e & 3));
      }
    }
    out[((size_t)rb * KC + kc) * 64 + lane] = b;
  }
}

size_t packed_q8_bytes(int M, int K) { return (size_t)((M + 15) / 16) * (K / 32) * 512; }

hipError_t launch_pack_q8(const uint16_t* W, int M, int K, void* out, float* scales, unsigned* bad, hipStream_t s) {
  if (K % 32) return hipErrorInvalidValue;
  pack_q8_kernel<<<(unsigned)((M + 15) / 16), 256, 0, s>>>(W, M, K, K / 32, (u32x2*)out, scales, bad);
  return hipGetLastError();
}

// A weight fragment slot as the A operand of v_mfma_f32_16x16x32_f16: the
// float16 copy as it is, or 8 codes plus 128 widened to float16.  Byte u is
// put under the exponent bits 0x64 (the float16 1024 + u, exact) and 1152 is
// subtracted (exact: u - 128 lies in [-128, 127]).
__device__ __forceinline__ f16x8 wfrag(const u32x4& w) { return __builtin_bit_cast(f16x8, w); }
__device__ __forceinline__ f16x8 wfrag(const u32x2& w) {
  u32x4 h;
  h[0] = __builtin_amdgcn_perm(0x64646464u, w[0], 0x04010400u);
  h[1] = __builtin_amdgcn_perm(0x64646464u, w[0], 0x04030402u);
  h[2] = __builtin_amdgcn_perm(0x64646464u, w[1], 0x04010400u);
  h[3] = __builtin_amdgcn_perm(0x64646464u, w[1], 0x04030402u);
  return __builtin_bit_cast(f16x8, h) - (f16x8)(_Float16)1152.0f;
}

// ------------------------------------------------------------------ GEMM, bf16 models (float16 operands)
//
// Y[n][o] = sum_k A[n][k] W[o][k] over packed weight fragments.
// A workgroup (4 waves) owns RB consecutive 16-row blocks and the k-steps
// [kc0, kc1) of its split (grid.y); wave w takes k-steps kc0 + w, kc0 + w + 4,
// ...  Per k-step a wave loads the RB weight fragments and the activation
// fragment of every node tile (float16, 1 KB contiguous each, see st_act)
// and multiplies each activation fragment into all RB row blocks, so
// activations are read once per RB row blocks.  U k-steps stay in flight
// (loads issued U steps ahead, unconditionally: a step past the end re-reads
// the last valid step and its weights are replaced by zeros when used), and
// scheduling barriers keep the compiler from sinking those loads next to
// their use.  After the loop the 4 waves are summed in wave order through
// LDS, so every output is computed the same way whatever the node count or a
// node's slot.
//  matrix cores: v_mfma_f32_16x16x32_f16, weight fragment as A (16 rows x 32
//    k), activations as B (32 k x 16 nodes);
//  vector ALU (few nodes): each lane multiplies its 8 weights into fp32
//    accumulators per node; the 4 lanes of a row are summed (xor 16, xor 32).
// Occupancy is traded for registers (1-2 waves per SIMD).
// Q8: 8-bit weight fragments (512 B), widened to float16 in registers before
// the product; each output is scaled by its row's scale before the epilogue.

template <int NT, int RB, int KIND, bool VEC, int NV, int U, int NW = 4, bool Q8 = false>
__global__ __launch_bounds__(64 * NW) __attribute__((amdgpu_waves_per_eu(NW / 4, NW / 2))) void gemm_kernel(
    const void* __restrict__ Wv, int KC, int RBtot, int kc_split, const uint16_t* __restrict__ act, Epi ep) {
  static_assert(!VEC || RB == 1, "vector path: one row block per workgroup");
  using WT = typename std::conditional<Q8, u32x2, u32x4>::type;
  const WT* Wp = (const WT*)Wv;
  constexpr int NB = VEC ? NV : NT;  // activation fragments per k-step
  constexpr int NN = VEC ? NV : 16 * NT;     // output nodes
  __shared__ float red[NW * RB * NN * 16];
  pass_signal(ep.sig);
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63;
  const int rb0 = blockIdx.x * RB;
  const int kc0 = blockIdx.y * kc_split;
  const int kc1 = min(KC, kc0 + kc_split);
  const int nsteps = kc1 - kc0 > w ? (kc1 - kc0 - w + NW - 1) / NW : 0;
  // weight rows past the matrix (last workgroup) read row block rb0 instead
  // and are never stored
  const WT* wb[RB];
#pragma unroll
  for (int r = 0; r < RB; ++r) wb[r] = Wp + (size_t)min(rb0 + r, RBtot - 1) * KC * 64 + lane;
  // activation fragments (see st_act): MFMA lanes read their own slot; in the
  // vector path lane l reads node n's slot in its 8-k group, 16 (l/16) + n
  const u32x4* abase = (const u32x4*)act + (VEC ? 16 * (lane >> 4) : lane);

  WT wq[U][RB];
  u32x4 bq[U][NB];
  const int klast = kc1 - 1;
  auto load_step = [&](int s, int u) {
    const int kc = min(kc0 + w + NW * s, klast);
#pragma unroll
    for (int r = 0; r < RB; ++r) wq[u][r] = wb[r][(size_t)kc * 64];
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      // b = node tile (matrix cores) or node (vector path)
      bq[u][b] = VEC ? abase[(size_t)kc * 64 + b] : abase[((size_t)b * KC + kc) * 64];
    }
  };

  f32x4 acc[RB][VEC ? 1 : NT];
  float vacc[VEC ? NV : 1];
#pragma unroll
  for (int r = 0; r < RB; ++r)
#pragma unroll
    for (int t = 0; t < (VEC ? 1 : NT); ++t) acc[r][t] = (f32x4){0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int n = 0; n < (VEC ? NV : 1); ++n) vacc[n] = 0.f;

  if (nsteps > 0) {
#pragma unroll
    for (int u = 0; u < U; ++u) load_step(u, u);
    __builtin_amdgcn_sched_barrier(0);
    for (int s0 = 0; s0 < nsteps; s0 += U) {
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int s = s0 + u;
        const bool ok = s < nsteps;
        if constexpr (!VEC) {
#pragma unroll
          for (int r = 0; r < RB; ++r) {
            const f16x8 wf = ok ? wfrag(wq[u][r]) : (f16x8)(_Float16)0.0f;
#pragma unroll
            for (int t = 0; t < NT; ++t)
              acc[r][t] = __builtin_amdgcn_mfma_f32_16x16x32_f16(wf, __builtin_bit_cast(f16x8, bq[u][t]),
                                                                 acc[r][t], 0, 0, 0);
          }
        } else {
          const f16x8 wf = ok ? wfrag(wq[u][0]) : (f16x8)(_Float16)0.0f;
          const f32x8 wv = __builtin_convertvector(wf, f32x8);
#pragma unroll
          for (int n = 0; n < NV; ++n) {
            const f32x8 av = __builtin_convertvector(__builtin_bit_cast(f16x8, bq[u][n]), f32x8);
#pragma unroll
            for (int e = 0; e < 8; ++e) vacc[n] = fmaf(wv[e], av[e], vacc[n]);
          }
        }
        __builtin_amdgcn_sched_barrier(0);
        load_step(s + U, u);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
  }

  // per-wave tiles -> LDS [wave][row block][node][16 rows], then the 4 waves summed in order
  if constexpr (!VEC) {
#pragma unroll
    for (int r = 0; r < RB; ++r)
#pragma unroll
      for (int t = 0; t < NT; ++t)
#pragma unroll
        for (int q = 0; q < 4; ++q)
          red[((w * RB + r) * NN + 16 * t + (lane & 15)) * 16 + 4 * (lane >> 4) + q] = acc[r][t][q];
  } else {
#pragma unroll
    for (int n = 0; n < NV; ++n) {
      float v = vacc[n];
      v += __shfl_xor(v, 16);
      v += __shfl_xor(v, 32);
      if (lane < 16) red[(w * NN + n) * 16 + lane] = v;
    }
  }
  __syncthreads();
  Epi e2 = ep;
  e2.split = blockIdx.y;
  for (int idx = tid; idx < RB * NN * 16; idx += 64 * NW) {
    const int row = idx & 15, node = (idx >> 4) % NN, r = idx / (16 * NN);
    const size_t st = (size_t)RB * NN * 16;
    const size_t base = ((size_t)r * NN + node) * 16 + row;
    float s = red[base];
#pragma unroll
    for (int ww = 1; ww < NW; ++ww) s += red[ww * st + base];
    const int o = (rb0 + r) * 16 + row;
    if (rb0 + r < RBtot && o < ep.M && node < ep.N) {
      if constexpr (Q8) s *= ep.wscale[o];
      epilogue<uint16_t, KIND>(e2, node, o, s);
    }
  }
}

// ------------------------------------------------------------------ weight GEMM for wide trees
//
// Above 64 nodes a workgroup of gemm_kernel reads every node's activations
// (N x K float16) for one or two row blocks of weights, so activation bytes
// dominate what each CU pulls in.  Here a workgroup owns RBT row blocks x
// kG2TT node tiles of the output over one k-range and reads RBT + kG2TT
// fragments per k-step.  Its four waves split the k-steps (wave w: kc0 + w,
// + 4, ...), each multiplying every weight fragment of a step into every
// activation fragment of it on v_mfma_f32_16x16x32_f16, and the waves'
// tiles are summed through LDS in wave order, one row block at a time.  The
// workgroups of one row-block group are placed on one XCD (workgroup b runs
// on XCD b % 8), so the weights they share come from HBM once and then from
// that XCD's L2.  Block b: XCD x = b % 8; q = b / 8 names (group i = x + 8
// (q / (gt gy)), node-tile group j, k-split sk); groups past gx exit.
constexpr int kG2TT = 4;  // node tiles per workgroup

template <int RBT, int KIND, int U, int NW, bool Q8>
__global__ __launch_bounds__(64 * NW) void gemm2d_kernel(const void* __restrict__ Wv, int KC, int RBtot, int NT,
                                                         int kcs, int gx, int gt, int gy,
                                                         const uint16_t* __restrict__ act, Epi ep) {
  constexpr int TT = kG2TT;
  using WT = typename std::conditional<Q8, u32x2, u32x4>::type;
  const WT* Wp = (const WT*)Wv;
  __shared__ float red[NW * TT * 16 * 16];
  pass_signal(ep.sig);
  const int b = blockIdx.x, x = b & 7, q = b >> 3, per = gt * gy;
  const int i = x + 8 * (q / per), rem = q % per;
  const int j = rem / gy, sk = rem % gy;
  if (i >= gx) return;
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63;
  const int rb0 = i * RBT, t0 = j * TT;
  const int kc0 = sk * kcs, kc1 = min(KC, kc0 + kcs);
  const int nsteps = kc1 - kc0 > w ? (kc1 - kc0 - w + NW - 1) / NW : 0;
  // row blocks past the matrix and node tiles past the tree read the last
  // one instead and are never stored
  const WT* wb[RBT];
  const u32x4* ab[TT];
#pragma unroll
  for (int r = 0; r < RBT; ++r) wb[r] = Wp + (size_t)min(rb0 + r, RBtot - 1) * KC * 64 + lane;
#pragma unroll
  for (int t = 0; t < TT; ++t) ab[t] = (const u32x4*)act + (size_t)min(t0 + t, NT - 1) * KC * 64 + lane;
  WT wq[U][RBT];
  u32x4 bq[U][TT];
  const int klast = kc1 - 1;
  auto load_step = [&](int s, int u) {
    const int kc = min(kc0 + w + NW * s, klast);
#pragma unroll
    for (int r = 0; r < RBT; ++r) wq[u][r] = wb[r][(size_t)kc * 64];
#pragma unroll
    for (int t = 0; t < TT; ++t) bq[u][t] = ab[t][(size_t)kc * 64];
  };
  f32x4 acc[RBT][TT];
#pragma unroll
  for (int r = 0; r < RBT; ++r)
#pragma unroll
    for (int t = 0; t < TT; ++t) acc[r][t] = (f32x4){0.f, 0.f, 0.f, 0.f};
  if (nsteps > 0) {
#pragma unroll
    for (int u = 0; u < U; ++u) load_step(u, u);
    __builtin_amdgcn_sched_barrier(0);
    for (int s0 = 0; s0 < nsteps; s0 += U) {
#pragma unroll
      for (int u = 0; u < U; ++u) {
        // (the step guard is uniform per wave: a select, never a branch
        // around an MFMA)
        const bool ok = s0 + u < nsteps;
#pragma unroll
        for (int r = 0; r < RBT; ++r) {
          const f16x8 wf = ok ? wfrag(wq[u][r]) : (f16x8)(_Float16)0.0f;
#pragma unroll
          for (int t = 0; t < TT; ++t)
            acc[r][t] = __builtin_amdgcn_mfma_f32_16x16x32_f16(wf, __builtin_bit_cast(f16x8, bq[u][t]), acc[r][t],
                                                               0, 0, 0);
        }
        __builtin_amdgcn_sched_barrier(0);
        load_step(s0 + u + U, u);
        __builtin_amdgcn_sched_barrier(0);
      }
    }
  }
  Epi e2 = ep;
  e2.split = sk;
#pragma unroll
  for (int r = 0; r < RBT; ++r) {
    if (rb0 + r >= RBtot) break;
    // lane l of a tile holds rows 4 (l / 16) + c, node l % 16
#pragma unroll
    for (int t = 0; t < TT; ++t)
#pragma unroll
      for (int c = 0; c < 4; ++c)
        red[((w * TT + t) * 16 + (lane & 15)) * 16 + 4 * (lane >> 4) + c] = acc[r][t][c];
    __syncthreads();
    for (int idx = tid; idx < TT * 256; idx += 64 * NW) {
      const int row = idx & 15, node = t0 * 16 + (idx >> 4);
      float sum = red[idx];
#pragma unroll
      for (int ww = 1; ww < NW; ++ww) sum += red[ww * TT * 256 + idx];
      const int o = (rb0 + r) * 16 + row;
      if (o < ep.M && node < ep.N) {
        if constexpr (Q8) sum *= ep.wscale[o];
        epilogue<uint16_t, KIND>(e2, node, o, sum);
      }
    }
    __syncthreads();
  }
}

// row blocks per workgroup of the wide-tree GEMM for a kind and node-tile
// group count: enough workgroups to cover the 256 CUs, as few activation
// re-reads as that allows (the LM head, with thousands of row blocks, takes 8)
static int g2_rbt(int kind, int gt) {
  if (kind == EPI_LOGITS) return 8;
  if (kind == EPI_PARTIAL) return gt <= 2 ? 1 : 2;
  return gt <= 2 ? 2 : 4;
}

bool gemm_wide(int vec, int N) { return !vec && N > 64; }

// Tile shape per node count and GEMM kind (measured on the GPT-2-L shapes:
// K = 1280 for QKV / MLP up / attention out, 5120 for MLP down).  At 17-32
// nodes: QKV one row block per workgroup (240 workgroups), the others two;
// 8 waves, with 1-5 k-steps of loads in flight.
GemmCfg gemm_cfg(int N, int vec, int kind) {
  GemmCfg c{};
  c.rb = 1;
  c.ck = 1;
  c.nw = 4;
  if (vec) {
    int nv = 1;
    while (nv < N) nv *= 2;
    c.nt = 1;
    c.nv = nv;
    return c;
  }
  int nt = 1;
  while (nt * 16 < N) nt *= 2;
  c.nt = nt;
  c.nv = 0;
  c.rb = nt <= 4 ? 2 : 1;
  if (nt == 2) {
    c.nw = 8;
    c.rb = kind == EPI_QKV ? 1 : 2;
  }
  return c;
}

int gemm_split_kc(int M, int K, int N, int vec, int want_split, int* splits) {
  const int KC = K / 32;
  if (!want_split) {
    *splits = 1;
    return KC;
  }
  if (gemm_wide(vec, N)) {
    const int gt = ((N + 15) / 16 + kG2TT - 1) / kG2TT;
    const int gx = ((M + 15) / 16 + g2_rbt(EPI_PARTIAL, gt) - 1) / g2_rbt(EPI_PARTIAL, gt);
    int S = 1;
    while (S * gx * gt < 256 && S < kMaxSplits) S *= 2;
    const int kcs = (KC + S - 1) / S;
    *splits = (KC + kcs - 1) / kcs;
    return kcs;
  }
  const int rb = gemm_cfg(N, vec, EPI_PARTIAL).rb;
  const int gx = ((M + 15) / 16 + rb - 1) / rb;
  int S = 1;  // a power of two with S * gx >= 256 workgroups
  while (S * gx < 256 && S < kMaxSplits) S *= 2;
  const int kcs = (KC + S - 1) / S;
  *splits = (KC + kcs - 1) / kcs;
  return kcs;
}

// row blocks per workgroup of the LM head (EPI_LOGITS on the matrix cores):
// it has thousands of row blocks, so more of them per workgroup make the
// activations (read once per workgroup) cost less than the weights
static int head_rb(int nt) { return nt <= 2 ? 8 : nt == 4 ? 4 : nt == 8 ? 2 : 1; }

GemmGeom gemm_geom(int kind, int vec, int M, int K, int N, int kcs) {
  GemmGeom g{};
  g.KC = K / 32;
  g.RBtot = (M + 15) / 16;
  g.kcs = kcs;
  if (gemm_wide(vec, N)) {
    // the wide-tree kernel as the prefetcher sees it: row-block groups
    // padded to a multiple of 8, so that group bx runs on XCD bx % 8 (plus
    // the launch's offset) like block bx of the plain kernel
    const int gt = ((N + 15) / 16 + kG2TT - 1) / kG2TT;
    g.RB = g2_rbt(kind, gt);
    g.gx = 8 * (((g.RBtot + g.RB - 1) / g.RB + 7) / 8);
    g.gy = (g.KC + kcs - 1) / kcs;
    return g;
  }
  if (vec) g.RB = 1;
  else if (kind == EPI_LOGITS) g.RB = head_rb(gemm_cfg(N, 0, kind).nt);
  else g.RB = gemm_cfg(N, 0, kind).rb;
  g.gx = (g.RBtot + g.RB - 1) / g.RB;
  g.gy = (g.KC + kcs - 1) / kcs;
  return g;
}

template <int NT, int RB, int KIND, bool VEC, int NV, int U, int NW = 4>
static void gemm_launch(const GemmGeom& g, const void* Wp, const uint16_t* act, const Epi& ep, hipStream_t s) {
  if (ep.wscale)
    gemm_kernel<NT, RB, KIND, VEC, NV, U, NW, true>
        <<<dim3(g.gx, g.gy), 64 * NW, 0, s>>>(Wp, g.KC, g.RBtot, g.kcs, act, ep);
  else
    gemm_kernel<NT, RB, KIND, VEC, NV, U, NW, false>
        <<<dim3(g.gx, g.gy), 64 * NW, 0, s>>>(Wp, g.KC, g.RBtot, g.kcs, act, ep);
}

template <int NT, int RB, bool VEC, int NV, int U>
static void gemm_go(int kind, const GemmGeom& g, const void* Wp, const uint16_t* act, const Epi& ep,
                    hipStream_t s) {
  switch (kind) {
    case EPI_QKV: gemm_launch<NT, RB, EPI_QKV, VEC, NV, U>(g, Wp, act, ep, s); break;
    case EPI_PARTIAL: gemm_launch<NT, RB, EPI_PARTIAL, VEC, NV, U>(g, Wp, act, ep, s); break;
    case EPI_GELU: gemm_launch<NT, RB, EPI_GELU, VEC, NV, U>(g, Wp, act, ep, s); break;
    default:
      if constexpr (VEC) gemm_launch<NT, RB, EPI_LOGITS, VEC, NV, U>(g, Wp, act, ep, s);
      break;
  }
}

template <int RBT, int KIND, int U, int NW>
static void gemm2d_launch(const dim3& grid, const void* Wp, int KC, int RBtot, int NT, int kcs, int gx, int gt,
                          int gy, const uint16_t* act, const Epi& ep, hipStream_t s) {
  if (ep.wscale)
    gemm2d_kernel<RBT, KIND, U, NW, true><<<grid, 64 * NW, 0, s>>>(Wp, KC, RBtot, NT, kcs, gx, gt, gy, act, ep);
  else
    gemm2d_kernel<RBT, KIND, U, NW, false><<<grid, 64 * NW, 0, s>>>(Wp, KC, RBtot, NT, kcs, gx, gt, gy, act, ep);
}

template <int RBT, int U, int NW>
static void gemm2d_go(int kind, const void* Wp, int KC, int RBtot, int NT, int kcs, int gx, int gt, int gy,
                      const uint16_t* act, const Epi& ep, hipStream_t s) {
  const dim3 grid(8 * ((gx + 7) / 8) * gt * gy);
  switch (kind) {
    case EPI_QKV: gemm2d_launch<RBT, EPI_QKV, U, NW>(grid, Wp, KC, RBtot, NT, kcs, gx, gt, gy, act, ep, s); break;
    case EPI_PARTIAL:
      gemm2d_launch<RBT, EPI_PARTIAL, U, NW>(grid, Wp, KC, RBtot, NT, kcs, gx, gt, gy, act, ep, s);
      break;
    case EPI_GELU: gemm2d_launch<RBT, EPI_GELU, U, NW>(grid, Wp, KC, RBtot, NT, kcs, gx, gt, gy, act, ep, s); break;
    default: gemm2d_launch<RBT, EPI_LOGITS, U, NW>(grid, Wp, KC, RBtot, NT, kcs, gx, gt, gy, act, ep, s); break;
  }
}

static hipError_t launch_gemm_wide(int kind, const void* Wp, int M, int K, const uint16_t* act, int kcs,
                                   const Epi& ep, hipStream_t s) {
  const int KC = K / 32, RBtot = (M + 15) / 16, NT = (ep.N + 15) / 16;
  const int gt = (NT + kG2TT - 1) / kG2TT, rbt = g2_rbt(kind, gt);
  const int gx = (RBtot + rbt - 1) / rbt, gy = (KC + kcs - 1) / kcs;
  if (kind != EPI_PARTIAL && gy != 1) return hipErrorInvalidValue;
  const void* W = Wp;
  switch (rbt) {
    case 1: gemm2d_go<1, 2, 4>(kind, W, KC, RBtot, NT, kcs, gx, gt, gy, act, ep, s); break;
    case 2: gemm2d_go<2, 2, 4>(kind, W, KC, RBtot, NT, kcs, gx, gt, gy, act, ep, s); break;
    case 4:
      // (QKV at more than 128 nodes: 8 waves, each with half the k-steps, measured
      // faster there; the other kinds and smaller trees are faster with 4)
      if (kind == EPI_QKV)
        gemm2d_launch<4, EPI_QKV, 2, 8>(dim3(8 * ((gx + 7) / 8) * gt * gy), W, KC, RBtot, NT, kcs, gx, gt, gy, act,
                                        ep, s);
      else
        gemm2d_go<4, 2, 4>(kind, W, KC, RBtot, NT, kcs, gx, gt, gy, act, ep, s);
      break;
    default: gemm2d_go<8, 1, 4>(kind, W, KC, RBtot, NT, kcs, gx, gt, gy, act, ep, s); break;
  }
  return hipGetLastError();
}

hipError_t launch_gemm_bf16(int kind, int vec, const void* Wp, int M, int K, const uint16_t* act, int kcs,
                            const Epi& ep, hipStream_t s) {
  if (kcs <= 0) return hipErrorInvalidValue;
  if (ep.N > (vec ? 16 : 256)) return hipErrorInvalidValue;
  if (gemm_wide(vec, ep.N)) return launch_gemm_wide(kind, Wp, M, K, act, kcs, ep, s);
  const GemmGeom g = gemm_geom(kind, vec, M, K, ep.N, kcs);
  if (kind == EPI_LOGITS && !vec) {
    switch (gemm_cfg(ep.N, 0, kind).nt) {
      case 1: gemm_launch<1, 8, EPI_LOGITS, false, 0, 3>(g, Wp, act, ep, s); break;
      case 2: gemm_launch<2, 8, EPI_LOGITS, false, 0, 2>(g, Wp, act, ep, s); break;
      case 4: gemm_launch<4, 4, EPI_LOGITS, false, 0, 2>(g, Wp, act, ep, s); break;
      case 8: gemm_launch<8, 2, EPI_LOGITS, false, 0, 1>(g, Wp, act, ep, s); break;
      default: gemm_launch<16, 1, EPI_LOGITS, false, 0, 1>(g, Wp, act, ep, s); break;
    }
    return hipGetLastError();
  }
  if (vec) {
    switch (gemm_cfg(ep.N, 1, kind).nv) {
      case 1: gemm_go<1, 1, true, 1, 8>(kind, g, Wp, act, ep, s); break;
      case 2: gemm_go<1, 1, true, 2, 8>(kind, g, Wp, act, ep, s); break;
      case 4: gemm_go<1, 1, true, 4, 6>(kind, g, Wp, act, ep, s); break;
      case 8: gemm_go<1, 1, true, 8, 4>(kind, g, Wp, act, ep, s); break;
      default: gemm_go<1, 1, true, 16, 2>(kind, g, Wp, act, ep, s); break;
    }
  } else {
    switch (gemm_cfg(ep.N, 0, kind).nt) {
      case 1: gemm_go<1, 2, false, 0, 6>(kind, g, Wp, act, ep, s); break;
      case 2:  // must match gemm_cfg
        if (kind == EPI_QKV) gemm_launch<2, 1, EPI_QKV, false, 0, 5, 8>(g, Wp, act, ep, s);
        else if (kind == EPI_GELU) gemm_launch<2, 2, EPI_GELU, false, 0, 3, 8>(g, Wp, act, ep, s);
        else gemm_launch<2, 2, EPI_PARTIAL, false, 0, 1, 8>(g, Wp, act, ep, s);
        break;
      case 4: gemm_go<4, 2, false, 0, 3>(kind, g, Wp, act, ep, s); break;
      case 8: gemm_go<8, 1, false, 0, 2>(kind, g, Wp, act, ep, s); break;
      default: gemm_go<16, 1, false, 0, 1>(kind, g, Wp, act, ep, s); break;
    }
  }
  return hipGetLastError();
}

// ------------------------------------------------------------------ weight prefetcher
//
// Runs on its own stream beside one pass (see PrefetchPlan).  Targets in
// order, per layer l: the QKV weights once MLP down of layer l - 1 (for
// l = 0: the embedding) has started, attention-out once the attention split
// has, MLP up once the attention merge has, MLP down once LN2 has; a target
// whose GEMM has itself started is skipped.  Block b (4 waves) on XCD x has
// rank b / 8 among the 32 blocks of its XCD and takes the GEMM blocks
// L = r + 8 j (r = (x - c) mod 8, c the XCD of the pass's block 0) with
// j = rank, rank + 32, ...; within one, wave w of nw loads k-steps w, w + nw, ... of
// each of its row blocks, kPfDepth fragments in flight, into registers folded
// into one value (stored only if it equals `magic`, so the loads are kept).
// The shallow depth paces the stream: the kernels running beside it are
// bound by memory latency, which a deeper burst raises by more than the warm
// weights save.  Thread 0 polls the signal counter with s_sleep between
// reads; every wait ends by the plan's timeout, after which the prefetcher
// stops.

constexpr int kPfBlocks = 256;
constexpr int kPfDepth = 4;

__global__ __launch_bounds__(256) void prefetcher_kernel(PrefetchPlan pp) {
  __shared__ int go;  // 1 prefetch, 0 skip, -1 stop
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63, nwv = blockDim.x >> 6;
  const int rank = blockIdx.x >> 3, nrank = gridDim.x >> 3;
  const unsigned x = xcc_id();
  const unsigned long long t0 = __builtin_amdgcn_s_memrealtime();
  unsigned acc = 0;
  for (int l = 0; l < pp.L; ++l) {
    for (int k = 0; k < 4; ++k) {
      const int target = k == 0 ? SIG_QKV : k == 1 ? SIG_OUT : k == 2 ? SIG_FC : SIG_PROJ;
      const int trig_k = k == 1 ? SIG_SPLIT : k == 2 ? SIG_MERGE : SIG_LN2;
      const unsigned long long trig =
          pp.base + (k == 0 ? (l == 0 ? 1 : sig_index(l - 1, SIG_PROJ)) : sig_index(l, trig_k));
      const unsigned long long late = pp.base + sig_index(l, target);
      if (tid == 0) {
        int v = -1;
        for (;;) {
          const unsigned long long p = __hip_atomic_load(pp.sig, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          if (p >= trig) {
            v = p >= late ? 0 : 1;
            break;
          }
          if (__builtin_amdgcn_s_memrealtime() - t0 > pp.timeout) break;
          __builtin_amdgcn_s_sleep(2);
        }
        go = v;
      }
      __syncthreads();
      const int g = go;
      __syncthreads();
      if (g < 0) {
        l = pp.L;
        break;
      }
      if (g == 0) continue;
      const unsigned c = __hip_atomic_load(pp.xcc0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      const int r = (int)((x - c) & 7u);
      const PfGeom G = pp.geo[k];
      typedef const __attribute__((address_space(1))) u32x4* gptr;  // global, not flat
      const gptr W = (gptr)pp.W[k * pp.L + l] + lane;
      const int J = G.nblk > r ? (G.nblk - r + 7) / 8 : 0;
      for (int j = rank; j < J; j += nrank) {
        const int L = r + 8 * j;
        const int bx = L % G.gx, by = L / G.gx;
        const int kc0 = by * G.kcs, nk = min(G.KC, kc0 + G.kcs) - kc0;
        for (int rr = 0; rr < G.RB; ++rr) {
          const gptr src = W + ((size_t)min(bx * G.RB + rr, G.RBtot - 1) * G.KC + kc0) * 64;
          for (int k0 = w; k0 < nk; k0 += nwv * kPfDepth) {
            u32x4 q[kPfDepth];
#pragma unroll
            for (int u = 0; u < kPfDepth; ++u) q[u] = src[(size_t)min(k0 + nwv * u, nk - 1) * 64];
#pragma unroll
            for (int u = 0; u < kPfDepth; ++u) acc ^= q[u][0] ^ q[u][1] ^ q[u][2] ^ q[u][3];
          }
        }
      }
    }
  }
  if (acc == pp.magic) *pp.sink = acc;
}

hipError_t launch_prefetcher(const PrefetchPlan& pp, hipStream_t s) {
  if (!pp.W || !pp.sig || !pp.xcc0 || !pp.sink || pp.L <= 0) return hipErrorInvalidValue;
  for (int k = 0; k < 4; ++k) {
    const PfGeom& G = pp.geo[k];
    if (G.KC <= 0 || G.RBtot <= 0 || G.RB <= 0 || G.kcs <= 0 || G.gx <= 0 || G.nblk <= 0 || G.nblk % G.gx)
      return hipErrorInvalidValue;
  }
  prefetcher_kernel<<<kPfBlocks, 256, 0, s>>>(pp);
  return hipGetLastError();
}

// ------------------------------------------------------------------ tree attention
//
// Node i, head h attends to cache rows 0..P-1 and then to its root path in the
// tree scratch (root first, itself last).  Two kernels:
//  prefix: workgroup (head h, tile s) stages cache rows 64s..64s+63 of head h
//    in LDS once and scores them against every node (one wave per node at a
//    time), leaving per (node, head, tile) the partial (max m, sum of exp z,
//    unnormalised output o[DH]);
//  combine: one wave per (node, head) merges the tiles' partials in tile order
//    with the node's root-path keys (read from the tree scratch) and writes
//    the normalised output into the next GEMM's input layout.
// Tiles are fixed by absolute key position, so a node's result does not
// depend on the other nodes.  Softmax in fp32; the 1/sqrt(head_dim) scale is
// applied to the dot products.

constexpr int ATT_WAVES = 16;

template <typename T, int DH>
__global__ __launch_bounds__(64 * ATT_WAVES) void attn_prefix_kernel(AttnArgs a) {
  constexpr int NT = 64 * ATT_WAVES;
  constexpr int EPU = 16 / sizeof(T);  // elements per 16-byte unit
  constexpr int UPR = DH / EPU;        // units per key row
  constexpr int TU = (64 * UPR + NT - 1) / NT;
  __shared__ float Ks[64][DH + 1];
  __shared__ float Vs[64][DH + 1];
  __shared__ float qs[64][DH];
  __shared__ float es[ATT_WAVES][64];
  const int h = blockIdx.x, s = blockIdx.y, tid = threadIdx.x, w = tid >> 6, lane = tid & 63;
  const int key0 = s * 64, nk = min(64, a.P - key0);
  const T* kc = (const T*)a.kc + ((size_t)h * a.max_ctx + key0) * DH;
  const T* vc = (const T*)a.vc + ((size_t)h * a.max_ctx + key0) * DH;
  {
    u32x4 kr[TU], vr[TU];
#pragma unroll
    for (int i = 0; i < TU; ++i) {
      const int idx = min(tid + i * NT, 64 * UPR - 1);
      const int j = min(idx / UPR, nk - 1), c = (idx % UPR) * EPU;
      kr[i] = *(const u32x4*)(kc + (size_t)j * DH + c);
      vr[i] = *(const u32x4*)(vc + (size_t)j * DH + c);
    }
#pragma unroll
    for (int i = 0; i < TU; ++i) {
      const int idx = tid + i * NT;
      if (idx < 64 * UPR) {
        const int j = idx / UPR, c = (idx % UPR) * EPU;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          if constexpr (sizeof(T) == 2) {
            Ks[j][c + 2 * e] = __uint_as_float(kr[i][e] << 16);
            Ks[j][c + 2 * e + 1] = __uint_as_float(kr[i][e] & 0xffff0000u);
            Vs[j][c + 2 * e] = __uint_as_float(vr[i][e] << 16);
            Vs[j][c + 2 * e + 1] = __uint_as_float(vr[i][e] & 0xffff0000u);
          } else {
            Ks[j][c + e] = __uint_as_float(kr[i][e]);
            Vs[j][c + e] = __uint_as_float(vr[i][e]);
          }
        }
      }
    }
  }
  for (int n0 = 0; n0 < a.N; n0 += 64) {
    const int nn = min(64, a.N - n0);
    __syncthreads();  // tile staged / previous node chunk done with qs
    for (int idx = tid; idx < 64 * DH / 4; idx += NT) {
      const int r = idx / (DH / 4), c = (idx % (DH / 4)) * 4;
      const float4 v4 = *(const float4*)(a.q + (size_t)(n0 + min(r, nn - 1)) * a.d + h * DH + c);
      qs[r][c] = v4.x;
      qs[r][c + 1] = v4.y;
      qs[r][c + 2] = v4.z;
      qs[r][c + 3] = v4.w;
    }
    __syncthreads();
    for (int r = w; r < nn; r += ATT_WAVES) {
      const int n = n0 + r;
      float dot = 0.f;
#pragma unroll 16
      for (int c = 0; c < DH; ++c) dot = fmaf(qs[r][c], Ks[lane][c], dot);
      const bool valid = lane < nk;
      const float sc = valid ? dot * a.scale : -INFINITY;
      const float m = wave_max(sc);
      const float e = valid ? expf(sc - m) : 0.f;
      const float z = wave_sum(e);
      es[w][lane] = e;
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
      float* out = a.part + (((size_t)h * a.S + s) * a.N + n) * (DH + 2);
      if (lane < DH) {
        float o = 0.f;
#pragma unroll 16
        for (int j = 0; j < 64; ++j) o = fmaf(es[w][j], Vs[j][lane], o);
        out[2 + lane] = o;
      }
      if (lane == 0) {
        out[0] = m;
        out[1] = z;
      }
      __builtin_amdgcn_wave_barrier();
    }
  }
}

template <typename T, int DH>
__global__ __launch_bounds__(256) void attn_combine_kernel(AttnArgs a) {
  constexpr int EPU = 16 / sizeof(T);
  const int pair = blockIdx.x * 4 + (threadIdx.x >> 6), lane = threadIdx.x & 63;
  if (pair >= a.N * a.H) return;
  const int n = pair / a.H, h = pair - n * a.H;
  float qv[DH];
#pragma unroll
  for (int c = 0; c < DH; c += 4) {
    const float4 t4 = *(const float4*)(a.q + (size_t)n * a.d + h * DH + c);
    qv[c] = t4.x;
    qv[c + 1] = t4.y;
    qv[c + 2] = t4.z;
    qv[c + 3] = t4.w;
  }
  const int dn = a.depth[n];
  const int* al = a.ancl + a.anc_off[n];
  const T* kt = (const T*)a.kt + (size_t)h * a.max_nodes * DH;
  const T* vt = (const T*)a.vt + (size_t)h * a.max_nodes * DH;
  const size_t pstride = (size_t)a.N * (DH + 2);  // between tiles
  const float* pp = a.part + ((size_t)h * a.S * a.N + n) * (DH + 2);

  // running (max, sum, output) over prefix tiles, then tree keys; values are
  // fetched 16 at a time (clamped) with every load issued before any use
  constexpr int B = 16;
  float m = -INFINITY, l = 0.f, o = 0.f;
  const int lc = min(lane, DH - 1);
  for (int s0 = 0; s0 < a.S; s0 += B) {
    const int cnt = min(B, a.S - s0);
    const int sl = s0 + min(lane, cnt - 1);
    const float ms0 = pp[(size_t)sl * pstride], zs0 = pp[(size_t)sl * pstride + 1];
    float ov[B];
#pragma unroll
    for (int j = 0; j < B; ++j) ov[j] = pp[(size_t)(s0 + min(j, cnt - 1)) * pstride + 2 + lc];
    const float ms = lane < cnt ? ms0 : -INFINITY;
    const float mn = fmaxf(m, wave_max(ms));
    const float alpha = expf(m - mn);
    const float ws = lane < cnt ? expf(ms - mn) : 0.f;
    l = l * alpha + wave_sum(lane < cnt ? zs0 * ws : 0.f);
    float acc = 0.f;
#pragma unroll
    for (int j = 0; j < B; ++j) acc = fmaf(ov[j], __shfl(ws, j), acc);
    o = o * alpha + acc;
    m = mn;
  }
  for (int t0 = 0; t0 <= dn; t0 += B) {
    const int cnt = min(B, dn + 1 - t0);
    const int t = t0 + min(lane, cnt - 1);
    const int key = al[t];
    float vv[B];
#pragma unroll
    for (int j = 0; j < B; ++j) vv[j] = ldT(vt, (size_t)__shfl(key, j) * DH + lc);
    float dot = 0.f;
    const T* kr = kt + (size_t)key * DH;
#pragma unroll
    for (int c = 0; c < DH; c += EPU) {
      const u32x4 ku = *(const u32x4*)(kr + c);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        if constexpr (sizeof(T) == 2) {
          dot = fmaf(qv[c + 2 * e], __uint_as_float(ku[e] << 16), dot);
          dot = fmaf(qv[c + 2 * e + 1], __uint_as_float(ku[e] & 0xffff0000u), dot);
        } else {
          dot = fmaf(qv[c + e], __uint_as_float(ku[e]), dot);
        }
      }
    }
    const bool valid = lane < cnt;
    const float sc = valid ? dot * a.scale : -INFINITY;
    const float mn = fmaxf(m, wave_max(sc));
    const float alpha = expf(m - mn);
    const float p = valid ? expf(sc - mn) : 0.f;
    l = l * alpha + wave_sum(p);
    float acc = 0.f;
#pragma unroll
    for (int j = 0; j < B; ++j) acc = fmaf(__shfl(p, j), vv[j], acc);
    o = o * alpha + acc;
    m = mn;
  }
  if (lane < DH) st_act((T*)a.out, n, h * DH + lane, a.ldo, o / l, a.err);
}

// ---- bf16 models: two kernels, the first on the matrix cores
//
// attn_split_kernel, block (head h, prefix chunk c) of CL cache rows, 8
//   waves.  The chunk's K rows and V^T are staged in LDS once (all its loads
//   in flight together, two per thread); wave w takes the 16-node tiles w,
//   w + 8, ... of the tree against them.  S^T = K Q^T and
//   O^T = V^T P^T run on v_mfma_f32_16x16x32_bf16 (q and p split into bf16
//   hi + lo, K and V exact) 32 keys at a time with an online softmax.  The K
//   operand's rows are ordered so that lane l ends up holding the scores of
//   keys 8(l/16)..+7 of node l%16, which is exactly its slot of the P^T
//   operand.  Each leaves a part (max, sum of exponentials, unnormalised
//   output) per (head, chunk, node).
// attn_merge_kernel: DH / 4 threads (four output dims each) per (node, head): the
//   chunks' parts merged in chunk order, then the node's root path (its
//   ancestors and itself in the tree scratch, root first) folded in RK keys
//   at a time, each score four products per thread then a butterfly sum
//   over the pair's threads; the output is written in the next GEMM's input
//   layout, four columns per store.  The chunking depends on P
//   only, so a node's result does not depend on the rest of the tree.

constexpr int AT_STAGE = kAttnMaxChunk;  // cache rows staged per block
constexpr int AT_MAXW = 8;               // waves per block

__device__ __forceinline__ void pack_hilo8(const float (&v)[8], u32x4& hi, u32x4& lo) {
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const uint32_t hp = f2bf2(v[2 * e], v[2 * e + 1]);
    hi[e] = hp;
    lo[e] = f2bf2(v[2 * e] - __uint_as_float(hp << 16), v[2 * e + 1] - __uint_as_float(hp & 0xffff0000u));
  }
}

__device__ __forceinline__ f32x4 mfma16(const u32x4& a, const u32x4& b, const f32x4& c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c, 0,
                                                  0, 0);
}

__device__ __forceinline__ void wave_sync_lds() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// a part record of the bf16 attention: max and sum of exponentials (float32),
// 8 bytes of padding, then the unnormalised output in float16 (it is rounded
// to float16 again as the next GEMM's input)
template <int DH> constexpr int part_bytes() { return 16 + 2 * DH; }
__device__ __forceinline__ uint32_t f16pair(float a, float b) {
  return (uint32_t)__builtin_bit_cast(uint16_t, (_Float16)a) | ((uint32_t)__builtin_bit_cast(uint16_t, (_Float16)b) << 16);
}

template <int DH>
__device__ __forceinline__ void attn_prefix_chunk(const AttnArgs& a, uint16_t* lds, int h, int c) {
  constexpr int KS = DH + 8;        // LDS row stride of K (elements)
  // LDS row stride of V^T (elements).  Row d holds key k at position
  // k ^ (8 ((d / 16) % 8)): the swizzle moves whole 8-key groups inside their
  // 32-key block (so an operand read of 8 keys stays one aligned 16-byte read,
  // and the 16 rows of one read share the swizzle), and it sends the staging
  // stores of one key's 64 dims, 8 rows apart, to different banks.
  constexpr int VS = AT_STAGE + 8;
  constexpr int MAXU = (AT_STAGE * DH / 8 + 64 * AT_MAXW - 1) / (64 * AT_MAXW);  // 16-byte units per thread
  uint16_t* ks = lds;
  uint16_t* vts = lds + AT_STAGE * KS;
  const int tid = threadIdx.x, nt = blockDim.x, nw = nt >> 6, w = tid >> 6, lane = tid & 63;
  const int i = lane & 15, g = lane >> 4;
  const int kbeg = c * a.CL, nk = min(a.CL, a.P - kbeg), nkr = (nk + 31) & ~31;
  const uint16_t* kc = (const uint16_t*)a.kc + ((size_t)h * a.max_ctx + kbeg) * DH;
  const uint16_t* vc = (const uint16_t*)a.vc + ((size_t)h * a.max_ctx + kbeg) * DH;
  const int units = nkr * (DH / 8);
  // the chunk's rows, all loads in flight at once (rows past the prefix
  // re-read the last row and are zeroed below)
  u32x4 kr[MAXU], vr[MAXU];
#pragma unroll
  for (int j = 0; j < MAXU; ++j) {
    const int e = tid + j * nt;
    if (e < units) {
      const int r = min(e / (DH / 8), nk - 1), c8 = e % (DH / 8);
      kr[j] = *(const u32x4*)(kc + (size_t)r * DH + 8 * c8);
      vr[j] = *(const u32x4*)(vc + (size_t)r * DH + 8 * c8);
    }
  }
  // queries of the wave's first tile (B operand: node 16 t + i, dims 32 kc2 + 8 g .. +8)
  const int ntiles = (a.N + 15) >> 4;
  f32x4 qf[DH / 32][2];
  auto load_q = [&](int t) {
    const int qn = min(16 * t + i, a.N - 1);
#pragma unroll
    for (int kc2 = 0; kc2 < DH / 32; ++kc2) {
      const float* qp = a.q + (size_t)qn * a.d + h * DH + 32 * kc2 + 8 * g;
      qf[kc2][0] = *(const f32x4*)qp;
      qf[kc2][1] = *(const f32x4*)(qp + 4);
    }
  };
  if (w < ntiles) load_q(w);
#pragma unroll
  for (int j = 0; j < MAXU; ++j) {
    const int e = tid + j * nt;
    if (e < units) {
      const int r = e / (DH / 8), c8 = e % (DH / 8);
      const bool ok = r < nk;
      const u32x4 kk = ok ? kr[j] : (u32x4){0, 0, 0, 0};
      const u32x4 vv = ok ? vr[j] : (u32x4){0, 0, 0, 0};
      const int vsw = 8 * ((c8 >> 1) & 7);  // V^T key swizzle of rows 8 c8 .. 8 c8 + 7
      *(u32x4*)(ks + r * KS + 8 * c8) = kk;
#pragma unroll
      for (int e2 = 0; e2 < 4; ++e2) {
        vts[(8 * c8 + 2 * e2) * VS + (r ^ vsw)] = (uint16_t)(vv[e2] & 0xffffu);
        vts[(8 * c8 + 2 * e2 + 1) * VS + (r ^ vsw)] = (uint16_t)(vv[e2] >> 16);
      }
    }
  }
  __syncthreads();
  const int ns = a.nsplit;
  for (int t = w; t < ntiles; t += nw) {
    if (t != w) load_q(t);
    u32x4 qh[DH / 32], ql[DH / 32];
#pragma unroll
    for (int kc2 = 0; kc2 < DH / 32; ++kc2) {
      const f32x4 f0 = qf[kc2][0], f1 = qf[kc2][1];
      const float v[8] = {f0[0], f0[1], f0[2], f0[3], f1[0], f1[1], f1[2], f1[3]};
      pack_hilo8(v, qh[kc2], ql[kc2]);
    }
    float m = -INFINITY, l = 0.f;
    f32x4 o[DH / 16];
#pragma unroll
    for (int tt = 0; tt < DH / 16; ++tt) o[tt] = (f32x4){0, 0, 0, 0};
    for (int sb = 0; sb < nkr / 32; ++sb) {
      // K operand rows: key 32 sb + 8 (i / 4) + i % 4 (+ 4 for s1)
      const uint16_t* kb = ks + (32 * sb + 8 * (i >> 2) + (i & 3)) * KS + 8 * g;
      f32x4 s0 = (f32x4){0, 0, 0, 0}, s1 = (f32x4){0, 0, 0, 0};
#pragma unroll
      for (int kc2 = 0; kc2 < DH / 32; ++kc2) {
        const u32x4 k0 = *(const u32x4*)(kb + 32 * kc2);
        const u32x4 k1 = *(const u32x4*)(kb + 4 * KS + 32 * kc2);
        s0 = mfma16(k0, qh[kc2], s0);
        s0 = mfma16(k0, ql[kc2], s0);
        s1 = mfma16(k1, qh[kc2], s1);
        s1 = mfma16(k1, ql[kc2], s1);
      }
      // lane: node 16 t + i, keys 32 sb + 8 g + e (e < 4 from s0, e >= 4 from s1)
      float sv[8];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int key = 32 * sb + 8 * g + r;
        sv[r] = key < nk ? s0[r] * a.scale : -INFINITY;
        sv[4 + r] = key + 4 < nk ? s1[r] * a.scale : -INFINITY;
      }
      float mb = sv[0];
#pragma unroll
      for (int e = 1; e < 8; ++e) mb = fmaxf(mb, sv[e]);
      mb = fmaxf(mb, __shfl_xor(mb, 16));
      mb = fmaxf(mb, __shfl_xor(mb, 32));
      const float mn = fmaxf(m, mb);
      const float alpha = __expf(m - mn);
      float pv[8], ps = 0.f;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        pv[e] = __expf(sv[e] - mn);
        ps += pv[e];
      }
      ps += __shfl_xor(ps, 16);
      ps += __shfl_xor(ps, 32);
      l = fmaf(l, alpha, ps);
      m = mn;
      u32x4 ph, pl;
      pack_hilo8(pv, ph, pl);
#pragma unroll
      for (int tt = 0; tt < DH / 16; ++tt) {
        const u32x4 va = *(const u32x4*)(vts + (16 * tt + i) * VS + ((32 * sb + 8 * g) ^ (8 * (tt & 7))));
        o[tt] = o[tt] * alpha;
        o[tt] = mfma16(va, ph, o[tt]);
        o[tt] = mfma16(va, pl, o[tt]);
      }
    }
    // part of node 16 t + i: lane (i, g) holds dims 16 tt + 4 g + r
    const int n = 16 * t + i;
    if (n < a.N) {
      unsigned char* rec = (unsigned char*)a.part + (((size_t)h * ns + c) * a.N + n) * part_bytes<DH>();
      if (g == 0) *(f32x2_t*)rec = (f32x2_t){m, l};
#pragma unroll
      for (int tt = 0; tt < DH / 16; ++tt)
        *(u32x2*)(rec + 16 + 2 * (16 * tt + 4 * g)) =
            (u32x2){f16pair(o[tt][0], o[tt][1]), f16pair(o[tt][2], o[tt][3])};
    }
  }
}

template <int DH>
__global__ __launch_bounds__(64 * AT_MAXW) void attn_split_kernel(AttnArgs a) {
  __shared__ __align__(16) uint16_t lds[AT_STAGE * (DH + 8) + DH * (AT_STAGE + 8)];  // K rows + V^T
  pass_signal(a.sig);
  // (an empty prefix launches one block, for the pass signal only)
  if ((int)blockIdx.x < a.H * a.nsplit) attn_prefix_chunk<DH>(a, lds, blockIdx.x % a.H, blockIdx.x / a.H);
}

// one wave per block: at 128 nodes x 20 heads that is 640 blocks, so every CU
// takes part (256-thread blocks left 96 of the 256 CUs idle)
constexpr int kMergeThreads = 64;

template <int DH>
__global__ __launch_bounds__(kMergeThreads) void attn_merge_kernel(AttnArgs a) {
  // TPP threads per (node, head), DPT = 4 consecutive dims each
  constexpr int RB = part_bytes<DH>(), DPT = 4, TPP = DH / DPT, PER = kMergeThreads / TPP, B = 16, RK = 8;
  pass_signal(a.sig);
  const int pair = blockIdx.x * PER + threadIdx.x / TPP, d0 = DPT * (threadIdx.x % TPP);
  if (pair >= a.N * a.H) return;  // (a whole pair's threads together)
  const int n = pair / a.H, h = pair - n * a.H, ns = a.nsplit;
  // the root path's first RK keys and these dims' query go out with the parts
  // (path32 is padded with the node itself, so every entry is a valid row)
  const int* p32 = a.path32 + (size_t)n * kPath32;
  const uint16_t* ktb = (const uint16_t*)a.kt + (size_t)h * a.max_nodes * DH + d0;
  const uint16_t* vtb = (const uint16_t*)a.vt + (size_t)h * a.max_nodes * DH + d0;
  const int rdep = a.depth[n];
  const f32x4 q4 = *(const f32x4*)(a.q + (size_t)n * a.d + h * DH + d0);
  int key[RK];
#pragma unroll
  for (int jj = 0; jj < RK; ++jj) key[jj] = p32[jj];
  const size_t cs = (size_t)a.N * RB;
  const unsigned char* rec = (const unsigned char*)a.part + ((size_t)h * ns * a.N + n) * RB;
  float M = -INFINITY, L = 0.f, O[DPT] = {0.f, 0.f, 0.f, 0.f};
  for (int c0 = 0; c0 < ns; c0 += B) {
    f32x2_t ml[B];
    u32x2 ov[B];
#pragma unroll
    for (int j = 0; j < B; ++j) {
      const int cc = min(c0 + j, ns - 1);
      ml[j] = *(const f32x2_t*)(rec + cc * cs);
      ov[j] = *(const u32x2*)(rec + cc * cs + 16 + 2 * d0);
    }
#pragma unroll
    for (int j = 0; j < B; ++j) {
      if (c0 + j >= ns) break;
      const float mn = fmaxf(M, ml[j][0]);
      const float al = __expf(M - mn), wj = __expf(ml[j][0] - mn);
      L = fmaf(L, al, ml[j][1] * wj);
      const float o4[DPT] = {h2f((uint16_t)(ov[j][0] & 0xffffu)), h2f((uint16_t)(ov[j][0] >> 16)),
                             h2f((uint16_t)(ov[j][1] & 0xffffu)), h2f((uint16_t)(ov[j][1] >> 16))};
#pragma unroll
      for (int e = 0; e < DPT; ++e) O[e] = fmaf(O[e], al, o4[e] * wj);
      M = mn;
    }
  }
  // the root path, root first, RK keys per batch
  for (int j0 = 0; j0 <= rdep; j0 += RK) {
    if (j0 > 0) {
#pragma unroll
      for (int jj = 0; jj < RK; ++jj) {
        const int j = min(j0 + jj, rdep);
        key[jj] = j < kPath32 ? p32[j] : a.ancl[a.anc_off[n] + j];
      }
    }
    u32x2 k4[RK], v4[RK];
#pragma unroll
    for (int jj = 0; jj < RK; ++jj) {
      k4[jj] = *(const u32x2*)(ktb + (size_t)key[jj] * DH);
      v4[jj] = *(const u32x2*)(vtb + (size_t)key[jj] * DH);
    }
    float s[RK];
#pragma unroll
    for (int jj = 0; jj < RK; ++jj)
      s[jj] = (q4[0] * __uint_as_float(k4[jj][0] << 16) + q4[1] * __uint_as_float(k4[jj][0] & 0xffff0000u)) +
              (q4[2] * __uint_as_float(k4[jj][1] << 16) + q4[3] * __uint_as_float(k4[jj][1] & 0xffff0000u));
    // (a butterfly leaves the same sum in every thread of the pair)
#pragma unroll
    for (int off = 1; off < TPP; off <<= 1)
#pragma unroll
      for (int jj = 0; jj < RK; ++jj) s[jj] += __shfl_xor(s[jj], off);
    float mb = -INFINITY;
#pragma unroll
    for (int jj = 0; jj < RK; ++jj) {
      s[jj] = j0 + jj <= rdep ? s[jj] * a.scale : -INFINITY;
      mb = fmaxf(mb, s[jj]);
    }
    const float mn = fmaxf(M, mb), al = __expf(M - mn);
    float ps = 0.f, po[DPT] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int jj = 0; jj < RK; ++jj) {
      const float p = __expf(s[jj] - mn);
      ps += p;
      const float v[DPT] = {__uint_as_float(v4[jj][0] << 16), __uint_as_float(v4[jj][0] & 0xffff0000u),
                            __uint_as_float(v4[jj][1] << 16), __uint_as_float(v4[jj][1] & 0xffff0000u)};
#pragma unroll
      for (int e = 0; e < DPT; ++e) po[e] = fmaf(p, v[e], po[e]);
    }
    L = fmaf(L, al, ps);
#pragma unroll
    for (int e = 0; e < DPT; ++e) O[e] = fmaf(O[e], al, po[e]);
    M = mn;
  }
  const float outv[DPT] = {O[0] / L, O[1] / L, O[2] / L, O[3] / L};
  st_act4_u16((uint16_t*)a.out, n, h * DH + d0, a.ldo, outv, a.err);
}

hipError_t launch_attn(int f32, int DH, const AttnArgs& a, hipStream_t s) {
  if (!f32) {
    if (a.N <= 0 || a.N > a.max_nodes || (DH != 64 && DH != 32)) return hipErrorInvalidValue;
    if (a.P > 0 && (a.CL <= 0 || a.CL > AT_STAGE || a.CL % 32 || a.nsplit != (a.P + a.CL - 1) / a.CL))
      return hipErrorInvalidValue;
    const int blocks = max(1, a.H * a.nsplit);
    const int mblocks = (a.N * a.H * (DH / 4) + kMergeThreads - 1) / kMergeThreads;
    if (DH == 64) {
      attn_split_kernel<64><<<blocks, 64 * AT_MAXW, 0, s>>>(a);
      attn_merge_kernel<64><<<mblocks, kMergeThreads, 0, s>>>(a);
    } else {
      attn_split_kernel<32><<<blocks, 64 * AT_MAXW, 0, s>>>(a);
      attn_merge_kernel<32><<<mblocks, kMergeThreads, 0, s>>>(a);
    }
    return hipGetLastError();
  }
  if (a.S > 0) {
    dim3 grid(a.H, a.S);
    const int nt = 64 * ATT_WAVES;
    if (DH == 64) attn_prefix_kernel<float, 64><<<grid, nt, 0, s>>>(a);
    else attn_prefix_kernel<float, 32><<<grid, nt, 0, s>>>(a);
  }
  const int blocks = (a.N * a.H + 3) / 4;
  if (DH == 64) attn_combine_kernel<float, 64><<<blocks, 256, 0, s>>>(a);
  else attn_combine_kernel<float, 32><<<blocks, 256, 0, s>>>(a);
  return hipGetLastError();
}

// ------------------------------------------------------------------ accept: greedy

// argmax of each logits row, lowest index among equal maxima
// greedy argmax per node (ties to the lowest token), in two stages so that
// the logits stream through many workgroups: chunks of kArgmaxChunk logits
// leave (value, index) pairs, then one wave per node merges its chunks
constexpr int kArgmaxChunk = 2048;

__device__ __forceinline__ bool better(float v, int i, float bv, int bi) { return v > bv || (v == bv && i < bi); }

__global__ __launch_bounds__(256) void argmax_part_kernel(const float* __restrict__ logits, int V, int C,
                                                          float* __restrict__ pv, int* __restrict__ pi) {
  __shared__ float sv[4];
  __shared__ int si[4];
  const int c = blockIdx.x, n = blockIdx.y, tid = threadIdx.x;
  const float* row = logits + (size_t)n * V;
  const int v0 = c * kArgmaxChunk;
  float x[kArgmaxChunk / 256];
#pragma unroll
  for (int k = 0; k < kArgmaxChunk / 256; ++k) x[k] = row[min(v0 + tid + 256 * k, V - 1)];
  float best = -INFINITY;
  int bi = V;
#pragma unroll
  for (int k = 0; k < kArgmaxChunk / 256; ++k) {
    const int v = v0 + tid + 256 * k;
    if (v < V && better(x[k], v, best, bi)) {
      best = x[k];
      bi = v;
    }
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    const float ov = __shfl_xor(best, off);
    const int oi = __shfl_xor(bi, off);
    if (better(ov, oi, best, bi)) {
      best = ov;
      bi = oi;
    }
  }
  if ((tid & 63) == 0) {
    sv[tid >> 6] = best;
    si[tid >> 6] = bi;
  }
  __syncthreads();
  if (tid == 0) {
    for (int w = 1; w < 4; ++w)
      if (better(sv[w], si[w], best, bi)) {
        best = sv[w];
        bi = si[w];
      }
    pv[(size_t)n * C + c] = best;
    pi[(size_t)n * C + c] = bi;
  }
}

__global__ __launch_bounds__(64) void argmax_final_kernel(const float* __restrict__ pv, const int* __restrict__ pi,
                                                          int V, int C, int* __restrict__ g) {
  const int n = blockIdx.x, lane = threadIdx.x;
  float best = -INFINITY;
  int bi = V;
  for (int c = lane; c < C; c += 64)
    if (better(pv[(size_t)n * C + c], pi[(size_t)n * C + c], best, bi)) {
      best = pv[(size_t)n * C + c];
      bi = pi[(size_t)n * C + c];
    }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    const float ov = __shfl_xor(best, off);
    const int oi = __shfl_xor(bi, off);
    if (better(ov, oi, best, bi)) {
      best = ov;
      bi = oi;
    }
  }
  if (lane == 0) g[n] = bi < V ? bi : 0;
}

// per-row top-k and log-sum-exp, in two stages like the argmax: chunks of
// kArgmaxChunk logits leave their top kTopKMax (value, index) pairs and
// (max, sum of exp(x - max)); one wave per row merges them.  A selection is
// k rounds of "best not yet taken" (ties to the lower index).
struct TopkPart {
  float v[kTopKMax];
  int i[kTopKMax];
  float m, s;
};

__global__ __launch_bounds__(256) void topk_part_kernel(const float* __restrict__ logits, int V, int C,
                                                        TopkPart* __restrict__ parts) {
  constexpr int E = kArgmaxChunk / 256;
  __shared__ float wv[4];
  __shared__ int wi[4];
  __shared__ float wm[4], wsum[4];
  const int c = blockIdx.x, n = blockIdx.y, tid = threadIdx.x, w = tid >> 6;
  const float* row = logits + (size_t)n * V;
  const int v0 = c * kArgmaxChunk;
  float x[E];
  unsigned taken = 0;
#pragma unroll
  for (int e = 0; e < E; ++e) {
    const int v = v0 + tid + 256 * e;
    x[e] = row[min(v, V - 1)];
    if (v >= V) taken |= 1u << e;
  }
  // chunk max and sum of exponentials (for the log-sum-exp)
  float mx = -INFINITY;
#pragma unroll
  for (int e = 0; e < E; ++e) mx = (taken >> e) & 1 ? mx : fmaxf(mx, x[e]);
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) mx = fmaxf(mx, __shfl_xor(mx, off));
  if ((tid & 63) == 0) wm[w] = mx;
  __syncthreads();
  mx = fmaxf(fmaxf(wm[0], wm[1]), fmaxf(wm[2], wm[3]));
  float se = 0.f;
#pragma unroll
  for (int e = 0; e < E; ++e) se += (taken >> e) & 1 ? 0.f : __expf(x[e] - mx);
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) se += __shfl_xor(se, off);
  if ((tid & 63) == 0) wsum[w] = se;
  TopkPart* out = parts + (size_t)n * C + c;
  for (int r = 0; r < kTopKMax; ++r) {
    // this thread's best untaken element (its elements are in increasing index order)
    float bv = -INFINITY;
    int bi = V, be = -1;
#pragma unroll
    for (int e = 0; e < E; ++e)
      if (!((taken >> e) & 1) && better(x[e], v0 + tid + 256 * e, bv, bi)) {
        bv = x[e];
        bi = v0 + tid + 256 * e;
        be = e;
      }
    float gv = bv;
    int gi = bi;
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
      const float ov = __shfl_xor(gv, off);
      const int oi = __shfl_xor(gi, off);
      if (better(ov, oi, gv, gi)) {
        gv = ov;
        gi = oi;
      }
    }
    __syncthreads();
    if ((tid & 63) == 0) {
      wv[w] = gv;
      wi[w] = gi;
    }
    __syncthreads();
    gv = wv[0];
    gi = wi[0];
    for (int k = 1; k < 4; ++k)
      if (better(wv[k], wi[k], gv, gi)) {
        gv = wv[k];
        gi = wi[k];
      }
    if (be >= 0 && gi == bi) taken |= 1u << be;
    if (tid == 0) {
      out->v[r] = gv;
      out->i[r] = gi;
    }
  }
  if (tid == 0) {
    out->m = mx;
    out->s = (wsum[0] + wsum[1]) + (wsum[2] + wsum[3]);
  }
}

__global__ __launch_bounds__(64) void topk_final_kernel(const TopkPart* __restrict__ parts, int V, int C, int k,
                                                        int* __restrict__ idx, float* __restrict__ val,
                                                        float* __restrict__ lse) {
  const int n = blockIdx.x, lane = threadIdx.x;
  const TopkPart* p = parts + (size_t)n * C;
  // log-sum-exp over the chunks in chunk order
  if (lane == 0 && lse) {
    float M = -INFINITY;
    for (int c = 0; c < C; ++c) M = fmaxf(M, p[c].m);
    float S = 0.f;
    for (int c = 0; c < C; ++c) S += p[c].s * __expf(p[c].m - M);
    lse[n] = M + logf(S);
  }
  // candidates: lane takes chunks lane, lane + 64, ...; each chunk's list is sorted
  // and a lane advances through its chunks' lists with one cursor per chunk
  constexpr int MAXC = 4;  // chunks per lane (vocab up to 64 * 4 * kArgmaxChunk)
  int cur[MAXC];
#pragma unroll
  for (int j = 0; j < MAXC; ++j) cur[j] = 0;
  for (int r = 0; r < k; ++r) {
    float bv = -INFINITY;
    int bi = V, bj = -1;
#pragma unroll
    for (int j = 0; j < MAXC; ++j) {
      const int c = lane + 64 * j;
      if (c < C && cur[j] < kTopKMax && better(p[c].v[cur[j]], p[c].i[cur[j]], bv, bi)) {
        bv = p[c].v[cur[j]];
        bi = p[c].i[cur[j]];
        bj = j;
      }
    }
    float gv = bv;
    int gi = bi;
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
      const float ov = __shfl_xor(gv, off);
      const int oi = __shfl_xor(gi, off);
      if (better(ov, oi, gv, gi)) {
        gv = ov;
        gi = oi;
      }
    }
    if (bj >= 0 && gi == bi) {
#pragma unroll
      for (int j = 0; j < MAXC; ++j)
        if (j == bj) ++cur[j];
    }
    if (lane == 0) {
      idx[(size_t)n * k + r] = gi < V ? gi : 0;
      val[(size_t)n * k + r] = gv;
    }
  }
}

size_t topk_work_bytes(int N, int V) {
  return (size_t)N * ((V + kArgmaxChunk - 1) / kArgmaxChunk) * sizeof(TopkPart);
}

hipError_t launch_topk(const float* logits, int N, int V, int k, int* idx, float* val, float* lse, void* work,
                       hipStream_t s) {
  const int C = (V + kArgmaxChunk - 1) / kArgmaxChunk;
  if (k < 1 || k > kTopKMax || C > 64 * 4) return hipErrorInvalidValue;
  TopkPart* parts = (TopkPart*)work;
  topk_part_kernel<<<dim3(C, N), 256, 0, s>>>(logits, V, C, parts);
  topk_final_kernel<<<N, 64, 0, s>>>(parts, V, C, k, idx, val, lse);
  return hipGetLastError();
}

// one thread: matched = parent matched and token == parent's argmax; keep the
// deepest matched node (lowest index among equals)
// The greedy walk over LDS copies of the tree (tok, par, dep) and the
// per-node argmax gl, by the whole block: node i is kept iff every edge on
// its root path has the child's token equal to its parent's argmax (pointer
// jumping: after round r, keep[i] covers the 2^r edges above i); the deepest
// kept node, the lowest index among equals, ends the path, and its argmax is
// the extra token.
__device__ void greedy_walk_lds(int N, const int* tok, const int* par, const int* dep, const int* gl, int* anc,
                                unsigned char* keep, int* redv, int* path, int* path_len, int* next) {
  const int tid = threadIdx.x, nt = blockDim.x;
  for (int i = tid; i < N; i += nt) {
    keep[i] = i == 0 || tok[i] == gl[par[i]];
    anc[i] = i == 0 ? -1 : par[i];
  }
  __syncthreads();
  for (int span = 1; span < N; span *= 2) {
    // (reads of the round complete before any write: two passes per round)
    unsigned char kv[4];
    int av[4];
    int c = 0;
    for (int i = tid; i < N && c < 4; i += nt, ++c) {
      const int a0 = anc[i];
      kv[c] = keep[i] && (a0 < 0 || keep[a0]);
      av[c] = a0 < 0 ? -1 : anc[a0];
    }
    __syncthreads();
    c = 0;
    for (int i = tid; i < N && c < 4; i += nt, ++c) {
      keep[i] = kv[c];
      anc[i] = av[c];
    }
    __syncthreads();
  }
  // deepest kept node, lowest index on ties: key = depth * 2^16 + (65535 - i)
  int best = 0;
  for (int i = tid; i < N; i += nt)
    if (keep[i]) best = max(best, (dep[i] << 16) | (65535 - i));
  for (int o = 32; o > 0; o >>= 1) best = max(best, __shfl_xor(best, o));
  if ((tid & 63) == 0) redv[tid >> 6] = best;
  __syncthreads();
  if (tid == 0) {
    int b = 0;
    for (int w = 0; w < nt / 64; ++w) b = max(b, redv[w]);
    const int bi = 65535 - (b & 65535);
    const int len = dep[bi] + 1;
    int j = bi;
    for (int t = len - 1; t >= 0; --t) {
      path[t] = j;
      j = par[j];
    }
    *path_len = len;
    *next = gl[bi];
  }
}

// greedy walk of up to 1024 nodes on the per-node argmax g (one block of
// 256 threads: each thread walks at most 4 nodes per pass)
__global__ __launch_bounds__(256) void greedy_walk_kernel(const int* __restrict__ tokens,
                                                          const int* __restrict__ parents,
                                                          const int* __restrict__ depth, int N,
                                                          const int* __restrict__ g, int* __restrict__ path,
                                                          int* __restrict__ path_len, int* __restrict__ next) {
  __shared__ int tok[1024], par[1024], dep[1024], gl[1024], anc[1024], redv[4];
  __shared__ unsigned char keep[1024];
  for (int i = threadIdx.x; i < N; i += blockDim.x) {
    tok[i] = tokens[i];
    par[i] = parents[i];
    dep[i] = depth[i];
    gl[i] = g[i];
  }
  __syncthreads();
  greedy_walk_lds(N, tok, par, dep, gl, anc, keep, redv, path, path_len, next);
}

// Greedy accept from per-workgroup maxima (the persistent pass's LM head
// leaves, for every node, each of G workgroups' largest logit and its token):
// 16 threads per node reduce its G pairs (ties to the lower token), then the
// block walks the tree as greedy_walk_kernel does.
__global__ __launch_bounds__(1024) void greedy_from_parts_kernel(const unsigned* __restrict__ parts, int G, int N,
                                                                  const int* __restrict__ tokens,
                                                                  const int* __restrict__ parents,
                                                                  const int* __restrict__ depth,
                                                                  int* __restrict__ path, int* __restrict__ path_len,
                                                                  int* __restrict__ next) {
  __shared__ int tok[64], par[64], dep[64], gl[64], anc[64], redv[16];
  __shared__ unsigned char keep[64];
  const int tid = threadIdx.x, n = tid >> 4, j = tid & 15;
  if (tid < N) {
    tok[tid] = tokens[tid];
    par[tid] = parents[tid];
    dep[tid] = depth[tid];
  }
  float v = -INFINITY;
  int o = 0x7fffffff;
  if (n < N) {
    // all of the thread's (up to 16) pairs loaded first, then compared
    typedef unsigned u2v __attribute__((ext_vector_type(2)));
    u2v pr[16];
#pragma unroll
    for (int q = 0; q < 16; ++q) {
      const int k = min(j + 16 * q, G - 1);
      pr[q] = *(const u2v*)(parts + ((size_t)n * G + k) * 2);
    }
#pragma unroll
    for (int q = 0; q < 16; ++q) {
      if (j + 16 * q >= G) break;
      const float v2 = __uint_as_float(pr[q].x);
      const int o2 = (int)pr[q].y;
      if (v2 > v || (v2 == v && o2 < o)) {
        v = v2;
        o = o2;
      }
    }
  }
#pragma unroll
  for (int msk = 1; msk < 16; msk <<= 1) {
    const float v2 = __shfl_xor(v, msk);
    const int o2 = __shfl_xor(o, msk);
    if (v2 > v || (v2 == v && o2 < o)) {
      v = v2;
      o = o2;
    }
  }
  if (j == 0 && n < N) gl[n] = o == 0x7fffffff ? 0 : o;  // (a row of NaN logits: token 0)
  __syncthreads();
  greedy_walk_lds(N, tok, par, dep, gl, anc, keep, redv, path, path_len, next);
}

hipError_t launch_greedy_from_parts(const unsigned* parts, int G, int N, const int* tokens, const int* parents,
                                    const int* depth, int* path, int* path_len, int* next, hipStream_t s) {
  if (N < 1 || N > 64 || G < 1 || G > 256) return hipErrorInvalidValue;
  greedy_from_parts_kernel<<<1, 1024, 0, s>>>(parts, G, N, tokens, parents, depth, path, path_len, next);
  return hipGetLastError();
}

size_t argmax_work_bytes(int N, int V) { return (size_t)N * ((V + kArgmaxChunk - 1) / kArgmaxChunk) * 8; }

hipError_t launch_argmax(const float* logits, int N, int V, int* g, void* work, hipStream_t s) {
  const int C = (V + kArgmaxChunk - 1) / kArgmaxChunk;
  float* pv = (float*)work;
  int* pi = (int*)(pv + (size_t)N * C);
  argmax_part_kernel<<<dim3(C, N), 256, 0, s>>>(logits, V, C, pv, pi);
  argmax_final_kernel<<<N, 64, 0, s>>>(pv, pi, V, C, g);
  return hipGetLastError();
}

hipError_t launch_greedy_walk(const int* tokens, const int* parents, const int* depth, int N, const int* g,
                              int* path, int* path_len, int* next, hipStream_t s) {
  if (N < 1 || N > 1024) return hipErrorInvalidValue;
  greedy_walk_kernel<<<1, 256, 0, s>>>(tokens, parents, depth, N, g, path, path_len, next);
  return hipGetLastError();
}

// ------------------------------------------------------------------ inverse-CDF picks
//
// For CDF-first tree assembly: query q draws from softmax(logits[rows[q]] / T)
// over the whole vocabulary at the uniform U[q] by inverse CDF in ascending
// token id.  One workgroup per query: thread t owns the contiguous ids
// [t C, t C + C); the row's maximum, then each thread's sum of the
// normalised probabilities in id order, then thread 0 walks the threads'
// sums in order to the crossing and scans that thread's ids (fp64
// throughout).  If rounding leaves no crossing, the last id with positive
// probability.
constexpr int kPickThreads = 1024;

__global__ __launch_bounds__(kPickThreads) void cdf_pick_kernel(CdfPickArgs a) {
  __shared__ double part[kPickThreads];
  __shared__ double red[kPickThreads / 64];
  const int q = blockIdx.x, tid = threadIdx.x, V = a.V;
  const float* row = a.logits + (size_t)a.rows[q] * V;
  const int C = (V + kPickThreads - 1) / kPickThreads, v0 = tid * C, v1 = min(V, v0 + C);
  double mx = -INFINITY;
  for (int v = v0; v < v1; ++v) mx = fmax(mx, (double)row[v] / a.T);
  for (int o = 32; o > 0; o >>= 1) mx = fmax(mx, __shfl_xor(mx, o));
  if ((tid & 63) == 0) red[tid >> 6] = mx;
  __syncthreads();
  if (tid == 0) {
    double m = red[0];
    for (int w = 1; w < kPickThreads / 64; ++w) m = fmax(m, red[w]);
    red[0] = m;
  }
  __syncthreads();
  mx = red[0];
  double e = 0.0;
  for (int v = v0; v < v1; ++v) e += exp((double)row[v] / a.T - mx);
  part[tid] = e;
  __syncthreads();
  if (tid == 0) {
    double S = 0.0;
    for (int t = 0; t < kPickThreads; ++t) S += part[t];
    red[1] = S;
  }
  __syncthreads();
  const double S = red[1];
  double c = 0.0;
  for (int v = v0; v < v1; ++v) c += exp((double)row[v] / a.T - mx) / S;
  __syncthreads();
  part[tid] = c;
  __syncthreads();
  if (tid == 0) {
    const double U = a.U[q];
    double run = 0.0;
    int pick = -1;
    for (int t = 0; t < kPickThreads && pick < 0; ++t) {
      if (run + part[t] > U) {
        double c3 = run;
        for (int v = t * C; v < min(V, t * C + C); ++v) {
          c3 += exp((double)row[v] / a.T - mx) / S;
          if (c3 > U) {
            pick = v;
            break;
          }
        }
      }
      run += part[t];
    }
    if (pick < 0) {
      pick = 0;
      for (int v = V - 1; v >= 0; --v)
        if (exp((double)row[v] / a.T - mx) / S > 0.0) {
          pick = v;
          break;
        }
    }
    a.out[q] = pick;
  }
}

hipError_t launch_cdf_pick(const CdfPickArgs& a, hipStream_t s) {
  if (a.n < 1 || a.n > kMaxPicks || a.V < 1 || !(a.T > 0.f)) return hipErrorInvalidValue;
  cdf_pick_kernel<<<a.n, kPickThreads, 0, s>>>(a);
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

// order-preserving key of a logit: a larger key is a larger value (-0 and
// +0 map to the same key, as they compare equal)
__device__ __forceinline__ unsigned mono_key(float f) {
  const unsigned u = __float_as_uint(f == 0.f ? 0.f : f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Recursive rejection sampling down the tree (Sec. 2.3 over the tree batch
// of Sec. 3.1), spread over G = ceil(V / 2048) workgroups: workgroup g holds
// the vocabulary slice [2048 g, 2048 g + 2048) of the current node's target
// p, residual r and draft row q in LDS (float64), thread t the 8 entries
// 8t .. 8t + 7 of the slice.  Every decision needs a few sums over the whole
// vocabulary; the workgroups exchange their slices' values in rounds: each
// stores a record, waits for its stores, raises its round flag, and waits
// for all G flags of the round, then reads every record and combines them
// in slice order, so all workgroups hold the same sums and take the same
// branches.  Records alternate between two buffers by round parity: a
// workgroup writes round k + 2 only after every workgroup has raised round
// k + 1, which each does after reading round k.
//
// Placement: 8 G workgroups are launched and those of index 8 g take slice
// g (the others leave at once), so that with the usual round-robin dispatch
// all G share one XCD.  The first round exchanges each workgroup's XCD; if
// they agree, later rounds keep records and flags in that XCD's L2 (plain
// stores; readers drop their CU's L1 first), otherwise every access is
// device-coherent (sc1) throughout.
//
// Rounds per node: the radix select of the top-k cut (4, plus 1 for the
// tie ranks), the softmax statistics (max, rescaled sum, draft sum: 1), then
// one per tested child: the owner of the child's token decides, and every
// workgroup adds up its slice's residual as it would be after a rejection;
// on rejection every workgroup applies it.  The extra token takes one more
// round (slice sums, then a scan of the crossing slice).
//
// Round flags carry epoch * 65536 + round, the epoch read from ctl[0] at
// start (the last workgroup to finish raises it), so nothing is cleared
// between calls.  Every wait is bounded; a wait that times out (the
// workgroups could not all run at once) raises ctl[2], every workgroup
// leaves, *path_len is set to 0 and err (when given) counts it.
// mode: 1 siblings drawn without replacement from draft row u, 2 drawn
// independently, 3 chosen (each child proposed with certainty; no draft
// rows), 4 CDF-first (no draft rows: the oracle's token at node u is the
// inverse CDF of its target at u's own uniform, stream 2, and the walk
// follows the first child carrying it; two rounds per node visited).
// topk > 0 restricts every target to the row's topk largest logits (ties at
// the cut to the lower id).

constexpr int SW_THREADS = 256, SW_SLICE = 2048, SW_PER = SW_SLICE / SW_THREADS, SW_MAXG = 64, SW_REC = 4;
constexpr int SW_MAXN = 1024;  // nodes (the tree's parents sit in LDS)
enum { SWC_EPOCH = 0, SWC_DONE = 1, SWC_ABORT = 2, SWC_FLAGS = 64 };
// work layout (bytes): ctl + flags (u32[SWC_FLAGS + SW_MAXG]), records
// double[2][SW_MAXG][SW_REC], histograms u32[2][SW_MAXG][256]
constexpr size_t kSwRecOfs = (SWC_FLAGS + SW_MAXG) * 4;
constexpr size_t kSwHistOfs = kSwRecOfs + (size_t)2 * SW_MAXG * SW_REC * 8;
constexpr size_t kSwBytes = kSwHistOfs + (size_t)2 * SW_MAXG * 256 * 4;

struct SwArgs {
  const int* tokens;
  const int* parents;
  int N, V, G;
  const float* logits;
  const float* draft;
  double T;
  uint64_t seed;
  int mode, topk;
  int* path;
  int* path_len;
  int* next;
  unsigned char* work;
  unsigned* err;
  unsigned long long timeout;
};

struct SwState {
  unsigned* ctl;
  unsigned* flags;
  double* rec;     // [2][SW_MAXG][SW_REC]
  unsigned* hist;  // [2][SW_MAXG][256]
  unsigned tagbase;
  int k;           // rounds done
  bool local;      // every workgroup on one XCD: records and flags through its L2
};

__device__ __forceinline__ unsigned sw_xcc() {
  unsigned x;
  asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(x));
  return x & 15;
}
__device__ __forceinline__ double* sw_rec(SwState& st, int par, int g) {
  return st.rec + ((size_t)par * SW_MAXG + g) * SW_REC;
}
__device__ __forceinline__ unsigned* sw_hist(SwState& st, int par, int g) {
  return st.hist + ((size_t)par * SW_MAXG + g) * 256;
}
// local: plain stores into the XCD's L2, read with non-temporal loads
// (which do not hit lines the reader's L1 kept from an earlier round);
// otherwise device-coherent (sc1) accesses
template <typename T>
__device__ __forceinline__ void sw_st(const SwState& st, T* p, T v) {
  if (st.local) *(__attribute__((address_space(1))) T*)p = v;
  else __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
template <typename T>
__device__ __forceinline__ T sw_ld(const SwState& st, const T* p) {
  if (st.local) return __builtin_nontemporal_load((const __attribute__((address_space(1))) T*)p);
  return __hip_atomic_load((T*)p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Fixed-order sums and maxima over the workgroup: each wave's value by a
// butterfly, lane 0's result taken (every lane then holds the same value),
// then the four waves in order; every thread returns the same value.
__device__ __forceinline__ double sw_wave_sum(double v) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return __shfl(v, 0);
}
__device__ __forceinline__ double sw_wave_max(double v) {
  for (int o = 32; o > 0; o >>= 1) v = fmax(v, __shfl_xor(v, o));
  return __shfl(v, 0);
}
__device__ void sw_sum2(double& a, double& b, double* red) {
  const double wa = sw_wave_sum(a), wb = sw_wave_sum(b);
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) {
    red[w] = wa;
    red[4 + w] = wb;
  }
  __syncthreads();
  a = (red[0] + red[1]) + (red[2] + red[3]);
  b = (red[4] + red[5]) + (red[6] + red[7]);
  __syncthreads();
}
__device__ double sw_max(double v, double* red) {
  const double wv = sw_wave_max(v);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = wv;
  __syncthreads();
  const double r = fmax(fmax(red[0], red[1]), fmax(red[2], red[3]));
  __syncthreads();
  return r;
}

// Publishes this workgroup's round (its record stores issued before) and
// waits for every workgroup's; false on abort or timeout (in every thread).
__device__ bool sw_round(const SwArgs& a, SwState& st, int g, int* shok) {
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  const unsigned tag = st.tagbase + (unsigned)st.k + 1u;
  if (threadIdx.x == 0) sw_st(st, st.flags + g, tag);
  if (threadIdx.x < 64) {
    const unsigned long long t0 = __builtin_amdgcn_s_memrealtime();
    bool ok = false;
    for (;;) {
      bool mine = true;
      for (int i = threadIdx.x; i < a.G; i += 64)
        mine = mine && (int)(__hip_atomic_load(st.flags + i, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) - tag) >= 0;
      if (__all(mine)) {
        ok = true;
        break;
      }
      if (__hip_atomic_load(st.ctl + SWC_ABORT, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) break;
      if (__builtin_amdgcn_s_memrealtime() - t0 > a.timeout) {
        if (threadIdx.x == 0 && __hip_atomic_exchange(st.ctl + SWC_ABORT, 1u, __ATOMIC_RELAXED,
                                                      __HIP_MEMORY_SCOPE_AGENT) == 0u && a.err)
          __hip_atomic_fetch_add(a.err, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        break;
      }
      __builtin_amdgcn_s_sleep(1);
    }
    if (threadIdx.x == 0) *shok = ok;
  }
  __syncthreads();
  const bool ok = *shok != 0;
  if (ok && st.local) asm volatile("buffer_inv sc0" ::: "memory");
  __syncthreads();
  ++st.k;
  return ok;
}

// every workgroup's record of round parity par into LDS (thread i loads
// workgroup i's), for the combining thread to read in slice order
__device__ __forceinline__ void sw_gather(SwState& st, int par, int G, double (*gb)[SW_REC]) {
  for (int i = threadIdx.x; i < G; i += SW_THREADS)
#pragma unroll
    for (int j = 0; j < SW_REC; ++j) gb[i][j] = sw_ld(st, sw_rec(st, par, i) + j);
  __syncthreads();
}

// the first child of u above index c0 (N if none): every thread tests its
// share of the candidates, then the smallest hit over the workgroup
__device__ __forceinline__ int sw_next_child(const int* par_l, int N, int u, int c0, int* shmin) {
  int best = N;
  for (int c = c0 + 1 + (int)threadIdx.x; c < N; c += SW_THREADS)
    if (par_l[c] == u) {
      best = c;
      break;
    }
  for (int o = 32; o > 0; o >>= 1) best = min(best, __shfl_xor(best, o));
  if ((threadIdx.x & 63) == 0) shmin[threadIdx.x >> 6] = best;
  __syncthreads();
  const int r = min(min(shmin[0], shmin[1]), min(shmin[2], shmin[3]));
  __syncthreads();
  return r;
}

// The smallest v whose running sum of w exceeds target, summed per thread
// in index order, per slice over threads in order, then over slices in order
// (if rounding leaves none, the last v with positive w), returned to every
// workgroup: one round for the slice sums, one for the pick of the slice's
// owner.  ok turns false (in every thread) on an abort or timeout.
__device__ int sw_pick_all(const SwArgs& a, SwState& st, int g, int G, const double* w, double target, int b0,
                           double* cs, double* red, double (*gb)[SW_REC], int* shi, bool& ok) {
  const int tid = threadIdx.x;
  double c1 = 0.0;
  int lastpos = -1;
#pragma unroll
  for (int i = 0; i < SW_PER; ++i) {
    const double wv = w[tid * SW_PER + i];
    c1 += wv;
    if (wv > 0.0) lastpos = b0 + i;
  }
  cs[tid] = c1;
  const int lp = (int)sw_max((double)lastpos, red);
  int par = st.k & 1;
  if (tid == 0) {
    double Wg = 0.0;
    for (int t = 0; t < SW_THREADS; ++t) Wg += cs[t];
    double* rc = sw_rec(st, par, g);
    sw_st(st, rc, Wg);
    sw_st(st, rc + 1, (double)lp);
  }
  ok = sw_round(a, st, g, shi + 1);
  if (!ok) return -1;
  sw_gather(st, par, G, gb);
  if (tid == 0) {
    double run = 0.0;
    int gx = -1, choice = -1;
    for (int gg = 0; gg < G; ++gg) {
      if (run + gb[gg][0] > target) {
        gx = gg;
        break;
      }
      run += gb[gg][0];
    }
    if (gx == g) {
      double c2 = run;
      for (int t = 0; t < SW_THREADS && choice < 0; ++t) {
        if (c2 + cs[t] > target) {
          double c3 = c2;
          for (int i = 0; i < SW_PER; ++i) {
            c3 += w[t * SW_PER + i];
            if (c3 > target) {
              choice = g * SW_SLICE + t * SW_PER + i;
              break;
            }
          }
        }
        c2 += cs[t];
      }
      if (choice < 0) choice = lp >= 0 ? lp : g * SW_SLICE;
    } else if (gx < 0) {
      // rounding left no crossing: the last token with positive weight
      choice = 0;
      for (int gg = G - 1; gg >= 0; --gg)
        if (gb[gg][1] >= 0.0) {
          choice = (int)gb[gg][1];
          break;
        }
    }
    shi[5] = gx;
    shi[6] = choice;
  }
  __syncthreads();
  const int gx = shi[5];
  if (gx < 0) {
    const int x = shi[6];
    __syncthreads();
    return x;
  }
  par = st.k & 1;
  if (tid == 0) sw_st(st, sw_rec(st, par, g), g == gx ? (double)shi[6] : 0.0);
  ok = sw_round(a, st, g, shi + 1);
  if (!ok) return -1;
  sw_gather(st, par, G, gb);
  const int x = (int)gb[gx][0];
  __syncthreads();
  return x;
}

__global__ __launch_bounds__(SW_THREADS) void sample_accept_kernel(SwArgs a) {
  if (blockIdx.x & 7) return;  // (see Placement above)
  __shared__ double r[SW_SLICE], p[SW_SLICE], q[SW_SLICE];
  __shared__ double red[8], cs[SW_THREADS];
  __shared__ unsigned hl[256];
  __shared__ int shi[8];
  __shared__ double shd[8];
  __shared__ double gb[SW_MAXG][SW_REC];
  __shared__ int par_l[SW_MAXN], shmin[4];
  const int tid = threadIdx.x, g = blockIdx.x >> 3, G = a.G, V = a.V;
  for (int i = tid; i < a.N; i += SW_THREADS) par_l[i] = a.parents[i];
  const int b0 = g * SW_SLICE + tid * SW_PER;  // this thread's first vocabulary index
  const bool wor = a.mode == 1, det = a.mode == 3, cdf = a.mode == 4;
  const bool cut = a.topk > 0 && a.topk < V;
  SwState st;
  st.ctl = (unsigned*)a.work;
  st.flags = st.ctl + SWC_FLAGS;
  st.rec = (double*)(a.work + kSwRecOfs);
  st.hist = (unsigned*)(a.work + kSwHistOfs);
  st.k = 0;
  st.local = false;
  if (tid == 0) shi[0] = (int)__hip_atomic_load(st.ctl + SWC_EPOCH, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  __syncthreads();
  st.tagbase = ((unsigned)shi[0] + 1u) * 65536u;
  // round 0: where every workgroup runs
  if (tid == 0) sw_st(st, sw_rec(st, 0, g), (double)sw_xcc());
  bool ok = sw_round(a, st, g, shi + 1);
  if (ok) {
    sw_gather(st, 0, G, gb);
    bool same = true;
    for (int i = 0; i < G; ++i) same = same && gb[i][0] == gb[0][0];
    st.local = same;
    __syncthreads();
  }
  int u = 0, len = 1, cdf_x = 0;
  if (ok && g == 0 && tid == 0) a.path[0] = 0;
  double Z = 1.0, Zq = 0.0;
  while (ok) {
    // ---- the target at node u: the thread's logits (and draft entries)
    float lg[SW_PER];
    unsigned key[SW_PER];
    bool keep[SW_PER];
#pragma unroll
    for (int i = 0; i < SW_PER; ++i) {
      const int v = b0 + i;
      lg[i] = v < V ? a.logits[(size_t)u * V + v] : 0.f;
      keep[i] = v < V;
      key[i] = mono_key(lg[i]);
      q[tid * SW_PER + i] = (!det && !cdf && v < V) ? (double)a.draft[(size_t)u * V + v] : 0.0;
    }
    if (cut) {
      // radix select of the topk-th largest key over all slices, 8 bits a pass
      unsigned prefix = 0, mask = 0;
      int need = a.topk;
      for (int pass = 0; pass < 4; ++pass) {
        const int shift = 24 - 8 * pass;
        hl[tid] = 0;
        __syncthreads();
#pragma unroll
        for (int i = 0; i < SW_PER; ++i)
          if (keep[i] && (key[i] & mask) == prefix) atomicAdd(&hl[(key[i] >> shift) & 255u], 1u);
        __syncthreads();
        const int par = st.k & 1;
        sw_st(st, sw_hist(st, par, g) + tid, hl[tid]);
        ok = sw_round(a, st, g, shi + 1);
        if (!ok) break;
        unsigned tot = 0;
        for (int gg = 0; gg < G; ++gg) tot += sw_ld(st, sw_hist(st, par, gg) + tid);
        hl[tid] = tot;
        __syncthreads();
        if (tid == 0) {
          int cum = 0, dgt = 255;
          for (; dgt > 0; --dgt) {
            if (cum + (int)hl[dgt] >= need) break;
            cum += (int)hl[dgt];
          }
          shi[2] = dgt;
          shi[3] = need - cum;
        }
        __syncthreads();
        prefix |= (unsigned)shi[2] << shift;
        mask |= 255u << shift;
        need = shi[3];
        __syncthreads();
      }
      if (!ok) break;
      // tie ranks at the cut: ties in lower slices, lower threads, then in order
      int cnt = 0;
#pragma unroll
      for (int i = 0; i < SW_PER; ++i) cnt += keep[i] && key[i] == prefix;
      cs[tid] = (double)cnt;
      __syncthreads();
      if (tid == 0) {
        double run = 0.0;
        for (int t = 0; t < SW_THREADS; ++t) {
          const double c = cs[t];
          cs[t] = run;
          run += c;
        }
        shd[0] = run;
      }
      __syncthreads();
      int rank = (int)cs[tid];
      const int par = st.k & 1;
      if (tid == 0) sw_st(st, sw_rec(st, par, g), shd[0]);
      ok = sw_round(a, st, g, shi + 1);
      if (!ok) break;
      sw_gather(st, par, G, gb);
      double base = 0.0;
      for (int gg = 0; gg < g; ++gg) base += gb[gg][0];
      rank += (int)base;
#pragma unroll
      for (int i = 0; i < SW_PER; ++i) {
        if (!keep[i] || key[i] > prefix) continue;
        keep[i] = key[i] == prefix && rank++ < need;
      }
    }
    // ---- softmax statistics over the kept entries, and the draft row's sum
    double mloc = -INFINITY;
#pragma unroll
    for (int i = 0; i < SW_PER; ++i)
      if (keep[i]) mloc = fmax(mloc, (double)lg[i] / a.T);
    const double m_g = sw_max(mloc, red);
    double sl = 0.0, ql = 0.0;
#pragma unroll
    for (int i = 0; i < SW_PER; ++i) {
      if (keep[i]) sl += exp((double)lg[i] / a.T - m_g);
      ql += q[tid * SW_PER + i];
    }
    sw_sum2(sl, ql, red);
    {
      const int par = st.k & 1;
      if (tid == 0) {
        double* rc = sw_rec(st, par, g);
        sw_st(st, rc, m_g);
        sw_st(st, rc + 1, sl);
        sw_st(st, rc + 2, ql);
      }
      ok = sw_round(a, st, g, shi + 1);
      if (!ok) break;
      sw_gather(st, par, G, gb);
      if (tid == 0) {
        double M = -INFINITY;
        for (int gg = 0; gg < G; ++gg) M = fmax(M, gb[gg][0]);
        double S = 0.0, Sq = 0.0;
        for (int gg = 0; gg < G; ++gg) {
          const double mg = gb[gg][0];
          if (mg != -INFINITY) S += gb[gg][1] * exp(mg - M);
          Sq += gb[gg][2];
        }
        shd[1] = M;
        shd[2] = S;
        shd[3] = Sq;
      }
      __syncthreads();
    }
    const double M = shd[1], S = shd[2];
    Zq = shd[3];
    __syncthreads();
#pragma unroll
    for (int i = 0; i < SW_PER; ++i) {
      const double pv = keep[i] ? exp((double)lg[i] / a.T - M) / S : 0.0;
      p[tid * SW_PER + i] = pv;
      r[tid * SW_PER + i] = pv;
    }
    __syncthreads();
    Z = 1.0;
    int accepted = -1;
    if (cdf) {
      // ---- the oracle's token at u: the inverse CDF of p at u's own
      // uniform; the walk follows the first child that carries it
      cdf_x = sw_pick_all(a, st, g, G, p, philox_uniform(a.seed, 2, (uint64_t)u), b0, cs, red, gb, shi, ok);
      if (!ok) break;
      for (int c = sw_next_child(par_l, a.N, u, u, shmin); c < a.N; c = sw_next_child(par_l, a.N, u, c, shmin))
        if (a.tokens[c] == cdf_x) {
          accepted = c;
          break;
        }
    }
    // ---- the children of u, in index order
    for (int c = cdf ? a.N : sw_next_child(par_l, a.N, u, u, shmin); c < a.N;
         c = sw_next_child(par_l, a.N, u, c, shmin)) {
      const int x = a.tokens[c];
      const int owner = x / SW_SLICE, xl = x - owner * SW_SLICE;
      // this slice's residual as it would be after rejecting x
      double zl = 0.0, zql = 0.0;
#pragma unroll
      for (int i = 0; i < SW_PER; ++i) {
        const int l = tid * SW_PER + i, v = b0 + i;
        double t;
        if (det) t = v == x ? 0.0 : r[l];
        else {
          const double dd = r[l] / Z - q[l] / Zq;
          t = dd > 0.0 ? dd : 0.0;
        }
        zl += t;
        zql += v == x ? 0.0 : q[l];
      }
      sw_sum2(zl, zql, red);
      const int par = st.k & 1;
      if (tid == 0) {
        double acc = 0.0;
        if (g == owner) {
          const double U = philox_uniform(a.seed, 0, (uint64_t)c);
          const double rx = r[xl];
          bool yes;
          if (det) {
            yes = Z > 0.0 && U < rx / Z;
          } else {
            const double qx = q[xl];
            yes = (qx == 0.0) ? (rx > 0.0) : (U < (rx / Z) / (qx / Zq));
          }
          acc = yes ? 1.0 : 0.0;
        }
        double* rc = sw_rec(st, par, g);
        sw_st(st, rc, zl);
        sw_st(st, rc + 1, zql);
        sw_st(st, rc + 2, acc);
      }
      ok = sw_round(a, st, g, shi + 1);
      if (!ok) break;
      sw_gather(st, par, G, gb);
      double zs = 0.0, zqs = 0.0;
      for (int gg = 0; gg < G; ++gg) {
        zs += gb[gg][0];
        zqs += gb[gg][1];
      }
      const bool yes = gb[owner][2] != 0.0;
      __syncthreads();  // (gb is rewritten by the next round's gather)
      if (yes) {
        accepted = c;
        break;
      }
      // rejected: apply the residual every workgroup summed
#pragma unroll
      for (int i = 0; i < SW_PER; ++i) {
        const int l = tid * SW_PER + i, v = b0 + i;
        if (det) {
          if (v == x) r[l] = 0.0;
        } else {
          const double dd = r[l] / Z - q[l] / Zq;
          r[l] = dd > 0.0 ? dd : 0.0;
          if (wor && v == x) q[l] = 0.0;
        }
      }
      Z = zs;
      if (wor) Zq = zqs;
      __syncthreads();
    }
    if (!ok || accepted < 0) break;
    if (g == 0 && tid == 0) a.path[len] = accepted;
    ++len;
    u = accepted;
    __syncthreads();
  }
  if (ok && cdf) {
    // ---- extra token: the oracle's token at the node the walk stopped at
    if (g == 0 && tid == 0) {
      *a.next = cdf_x;
      *a.path_len = len;
    }
  } else if (ok) {
    // ---- extra token: the smallest v whose running sum of w exceeds U2 * Z
    // (w = r, or p when rounding left no residual mass), summed per thread in
    // index order, per slice over threads in order, then over slices in order
    const double U2 = philox_uniform(a.seed, 1, (uint64_t)u);
    const bool use_r = Z > 0.0;
    const double* w = use_r ? r : p;
    const double target = U2 * (use_r ? Z : 1.0);
    double c1 = 0.0;
    int lastpos = -1;
#pragma unroll
    for (int i = 0; i < SW_PER; ++i) {
      const double wv = w[tid * SW_PER + i];
      c1 += wv;
      if (wv > 0.0) lastpos = b0 + i;
    }
    cs[tid] = c1;
    const int lp = (int)sw_max((double)lastpos, red);
    const int par = st.k & 1;
    if (tid == 0) {
      double Wg = 0.0;
      for (int t = 0; t < SW_THREADS; ++t) Wg += cs[t];
      double* rc = sw_rec(st, par, g);
      sw_st(st, rc, Wg);
      sw_st(st, rc + 1, (double)lp);
    }
    ok = sw_round(a, st, g, shi + 1);
    if (ok) sw_gather(st, par, G, gb);
    if (ok && tid == 0) {
      // the slice where the running sum crosses the target
      double run = 0.0;
      int gx = -1;
      for (int gg = 0; gg < G; ++gg) {
        if (run + gb[gg][0] > target) {
          gx = gg;
          break;
        }
        run += gb[gg][0];
      }
      int choice = -1;
      if (gx == g) {
        // in it, the thread chunk, then the entry
        double c2 = run;
        for (int t = 0; t < SW_THREADS && choice < 0; ++t) {
          if (c2 + cs[t] > target) {
            double c3 = c2;
            for (int i = 0; i < SW_PER; ++i) {
              c3 += w[t * SW_PER + i];
              if (c3 > target) {
                choice = g * SW_SLICE + t * SW_PER + i;
                break;
              }
            }
          }
          c2 += cs[t];
        }
        if (choice < 0) choice = lp >= 0 ? lp : g * SW_SLICE;  // rounding left no crossing in the slice
      } else if (gx < 0 && g == 0) {
        // rounding left no crossing: the last token with positive weight
        choice = 0;
        for (int gg = G - 1; gg >= 0; --gg)
          if (gb[gg][1] >= 0.0) {
            choice = (int)gb[gg][1];
            break;
          }
      }
      if (choice >= 0) *a.next = choice;
      if (g == 0) *a.path_len = len;
    }
  }
  // the last workgroup out raises the epoch (and clears an abort)
  __syncthreads();
  if (tid == 0) {
    if (!ok && g == 0) *a.path_len = 0;
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    const unsigned prev = __hip_atomic_fetch_add(st.ctl + SWC_DONE, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (prev == (unsigned)G - 1) {
      __hip_atomic_store(st.ctl + SWC_DONE, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(st.ctl + SWC_ABORT, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(st.ctl + SWC_EPOCH, (st.tagbase >> 16), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
}

static_assert(kSwBytes == kSampleWorkBytes, "the exchange area's size is declared in ssd_internal.h");
size_t sample_work_bytes() { return kSwBytes; }

hipError_t launch_sample_accept(const int* tokens, const int* parents, int N, int V, const float* logits,
                                const float* draft, double temperature, uint64_t seed, int mode, int topk, void* work,
                                unsigned* err, int* path, int* path_len, int* next, hipStream_t s) {
  if (mode < 1 || mode > 4 || (mode >= 3) != (draft == nullptr)) return hipErrorInvalidValue;
  const int G = (V + SW_SLICE - 1) / SW_SLICE;
  if (V <= 0 || G > SW_MAXG || N <= 0 || N > SW_MAXN || !work) return hipErrorInvalidValue;
  SwArgs a{tokens, parents, N, V, G, logits, draft, temperature, seed, mode, topk, path, path_len, next,
           (unsigned char*)work, err, 50000000ull /* 0.5 s at 100 MHz */};
  sample_accept_kernel<<<8 * G, SW_THREADS, 0, s>>>(a);
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
