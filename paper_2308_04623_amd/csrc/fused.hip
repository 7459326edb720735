// The whole verification pass of a bfloat16 model (head dimension 64, at most
// 64 tree nodes) as one persistent launch on CDNA4 (gfx950).
//
// Sec. 2.1 of Spector & Re (arXiv 2308.04623) observes that one small-batch
// decode step of a transformer is bound by streaming the weights from memory,
// and Sec. 3.1 makes the step score a whole token tree against the cached
// prefix.  At GPT-2-L size each layer's four weight matrices take about 6 us
// to stream at full HBM bandwidth, so the pass cannot afford a kernel boundary
// (3-7 us each) per sub-layer.  Here one launch runs every layer:
//
//  * 256 compute workgroups, one per CU.  A workgroup reads the XCD it runs
//    on from the hardware (x) and takes rank r = blockIdx / 8 within it.  Each
//    XCD owns a contiguous range of heads and a slice of the MLP's hidden
//    features, sized so that every XCD streams the same weight bytes per
//    layer.  Inside an XCD the work of a stage is split over its 32 ranks
//    (see the host planner below).
//  * Stages per layer: LN1 (residual update + LayerNorm of the XCD's rows),
//    QKV (the XCD's heads), ATT (tree attention per head and 16-node tile),
//    WO (attention out-projection over the XCD's heads: a partial residual),
//    LN2, FC (+GELU, the XCD's hidden slice), WPR (MLP down-projection over
//    that slice: a partial residual).  Only the two partial residuals cross
//    XCDs: every XCD adds its partial of each output, in fixed point (units
//    of 2^-32, 64-bit integers), into one device-wide sum with an atomic add;
//    integer addition does not depend on the order the XCDs arrive in, so
//    every XCD reads the same sum, adds it to its own copy of the residual
//    stream, and all copies agree bit for bit.  Every other hand-off stays
//    inside one XCD's L2.
//  * Inside a workgroup (8 waves): waves 4..7 run a stage's GEMM and issue
//    their first weight loads before its dependency is met; waves 0..3 run
//    the LayerNorm rows of the stage before it, and then wave 0 alone polls
//    for the dependency.  A CU returns vector loads in issue order, across
//    its waves, so the polling wave keeps nothing of its own in flight; a
//    poll still waits behind the other waves' loads.  With two or more node
//    tiles, waves 1..3 also copy into LDS the weights of a GEMM two stages
//    on: the out-projection's during LN1 + QKV, and the down-projection's
//    during the up-projection (at four tiles already during LN2's wait).
//  * Hand-offs are per-workgroup stage flags carrying a monotonically
//    increasing tag (pass, layer, stage).  A workgroup writes its outputs,
//    waits for its stores, then stores its flag; consumers poll the 32 flags
//    of their XCD or all 256 flags.  Data and flags read across XCDs use
//    device-coherent (sc1) accesses; inside an XCD plain stores, and loads
//    after the waiting wave dropped its CU's L1 lines, suffice.
//  * Every wait is bounded (s_memrealtime); a timeout raises an abort word
//    that every other wait also watches, so all workgroups leave the kernel,
//    and the session's error counter records it.
//
// Arithmetic per output is fixed by the matrix, the k-range of the XCD and
// the workgroup-internal split, never by the node count or a node's slot, so
// a node's logits do not depend on the rest of the tree.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include <algorithm>
#include <string>
#include <type_traits>
#include <vector>

#include "ssd_internal.h"

namespace ssd {
namespace fz {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x8 __attribute__((ext_vector_type(8)));
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef unsigned u32x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(3))) float lds_f32;
typedef __attribute__((address_space(3))) f32x4 lds_f32x4;
typedef float f32x2_t __attribute__((ext_vector_type(2)));

// A weight fragment slot as the A operand of v_mfma_f32_16x16x32_f16: the
// float16 copy as it is, or (8-bit models) 8 codes plus 128 widened to
// float16: byte u goes under the exponent bits 0x64 (the float16 1024 + u,
// exact) and 1152 is subtracted (exact: u - 128 lies in [-128, 127]).
__device__ __forceinline__ f16x8 wfrag(const u32x4& w) { return __builtin_bit_cast(f16x8, w); }
__device__ __forceinline__ f16x8 wfrag(const u32x2& w) {
  u32x4 h;
  h[0] = __builtin_amdgcn_perm(0x64646464u, w[0], 0x04010400u);
  h[1] = __builtin_amdgcn_perm(0x64646464u, w[0], 0x04030402u);
  h[2] = __builtin_amdgcn_perm(0x64646464u, w[1], 0x04010400u);
  h[3] = __builtin_amdgcn_perm(0x64646464u, w[1], 0x04030402u);
  return __builtin_bit_cast(f16x8, h) - (f16x8)(_Float16)1152.0f;
}

// Global-memory pointers (address space 1): loads through them are
// global_load, waited on in order, never flat.
template <typename T>
using gptr = const __attribute__((address_space(1))) T*;
template <typename T>
using gw = __attribute__((address_space(1))) T*;
template <typename T>
__device__ __forceinline__ gptr<T> G(const void* p) {
  return (gptr<T>)p;
}

constexpr int NTH = 512;  // threads per workgroup
constexpr int NWV = NTH / 64;  // waves per workgroup
constexpr int DH = 64;

__device__ __forceinline__ float bf2f(uint16_t h) { return __uint_as_float((uint32_t)h << 16); }
__device__ __forceinline__ uint16_t f2bf(float f) { return __builtin_bit_cast(uint16_t, (__bf16)f); }
__device__ __forceinline__ uint32_t f2bf2(float a, float b) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t){a, b}, bf16x2_t));
}
__device__ __forceinline__ unsigned xcc_id() {
  unsigned x;
  asm volatile("s_getreg_b32 %0, hwreg(HW_REG_XCC_ID)" : "=s"(x));
  return x & 15;
}
__device__ __forceinline__ unsigned long long now() { return __builtin_amdgcn_s_memrealtime(); }

// float16 GEMM input in matrix-core fragment order (ld = k-steps of 32 per
// 16-node tile): element (n, k) in fragment (n/16) ld + k/32, lane
// (n%16) + 16 ((k%32)/8), position k%8.  A value past float16's range
// (|v| > 65504, or NaN) would enter the matrix cores as inf or NaN: it is
// counted in err (the session's error counter) and stored as converted.
// (one count per wave and call: the lowest lane out of range adds 1)
__device__ __forceinline__ void f16_range(float v, unsigned* err) {
  const bool over = !(fabsf(v) <= 65504.f);
  const unsigned long long m = __builtin_amdgcn_ballot_w64(over);
  if (m && (int)__builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, 0u)) == __builtin_ctzll(m))
    __hip_atomic_fetch_add(err, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ void st_act(gw<uint16_t> p, int n, int k, int ld, float v, unsigned* err) {
  const size_t f = (size_t)(n >> 4) * ld + (k >> 5);
  f16_range(v, err);
  p[f * 512 + ((n & 15) + 16 * ((k & 31) >> 3)) * 8 + (k & 7)] = __builtin_bit_cast(uint16_t, (_Float16)v);
}

// four consecutive elements (n, k .. k+3), k % 4 == 0: one 8-byte store
__device__ __forceinline__ void st_act4(gw<uint16_t> p, int n, int k, int ld, float v0, float v1, float v2, float v3,
                                        unsigned* err) {
  const size_t f = (size_t)(n >> 4) * ld + (k >> 5);
  f16_range(fmaxf(fmaxf(fabsf(v0), fabsf(v1)), fmaxf(fabsf(v2), fabsf(v3))) + (v0 + v1 + v2 + v3) * 0.f, err);
  const uint32_t lo = (uint32_t)__builtin_bit_cast(uint16_t, (_Float16)v0) |
                      ((uint32_t)__builtin_bit_cast(uint16_t, (_Float16)v1) << 16);
  const uint32_t hi = (uint32_t)__builtin_bit_cast(uint16_t, (_Float16)v2) |
                      ((uint32_t)__builtin_bit_cast(uint16_t, (_Float16)v3) << 16);
  *(gw<u32x2>)(p + f * 512 + ((n & 15) + 16 * ((k & 31) >> 3)) * 8 + (k & 7)) = (u32x2){lo, hi};
}

constexpr int CP_SC1 = 16;  // cache policy of a device-coherent load (sc1)

__device__ __forceinline__ float gelu_tanh(float x) {
  const float c = 0.7978845608028654f;  // sqrt(2/pi)
  return 0.5f * x * (1.0f + tanhf(c * (x + 0.044715f * x * x * x)));
}

__device__ __forceinline__ void pack_hilo8(const float (&v)[8], u32x4& hi, u32x4& lo) {
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const uint32_t hp = f2bf2(v[2 * e], v[2 * e + 1]);
    hi[e] = hp;
    lo[e] = f2bf2(v[2 * e] - __uint_as_float(hp << 16), v[2 * e + 1] - __uint_as_float(hp & 0xffff0000u));
  }
}

__device__ __forceinline__ f32x4 mfma_bf16(const u32x4& a, const u32x4& b, const f32x4& c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c, 0,
                                                  0, 0);
}

__device__ __forceinline__ void wave_sync_lds() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}


// A uniform base pointer the compiler must treat as new at each use, so that
// per-thread addresses derived from it are formed inside the stage body
// instead of being hoisted out of the stage loop (where they would occupy,
// and spill, registers for the whole pass).
__device__ __forceinline__ unsigned long long opq_bits(unsigned long long v) {
  unsigned lo = __builtin_amdgcn_readfirstlane((unsigned)v), hi = __builtin_amdgcn_readfirstlane((unsigned)(v >> 32));
  asm volatile("" : "+s"(lo), "+s"(hi));
  return ((unsigned long long)hi << 32) | lo;
}
// the thread index, opaque for the same reason
__device__ __forceinline__ int opq_tid() {
  int t = threadIdx.x;
  asm volatile("" : "+v"(t));
  return t;
}
template <class T>
__device__ __forceinline__ gw<T> opq(T* p) {
  return (gw<T>)opq_bits((unsigned long long)p);
}
template <class T>
__device__ __forceinline__ gptr<T> opq(const T* p) {
  return (gptr<T>)opq_bits((unsigned long long)p);
}
template <class T>
__device__ __forceinline__ gptr<T> opq(gptr<T> p) {
  return (gptr<T>)opq_bits((unsigned long long)p);
}

// loads of data another CU of this XCD wrote during the pass: miss the L1
__device__ __forceinline__ u32x4 ld_x(const u32x4* p) { return __builtin_nontemporal_load(p); }
__device__ __forceinline__ float ld_x(const float* p) { return __builtin_nontemporal_load(p); }
__device__ __forceinline__ int ld_x(const int* p) { return __builtin_nontemporal_load(p); }
__device__ __forceinline__ u32x4 ld_x(gptr<u32x4> p) { return __builtin_nontemporal_load(p); }
__device__ __forceinline__ float ld_x(gptr<float> p) { return __builtin_nontemporal_load(p); }
__device__ __forceinline__ int ld_x(gptr<int> p) { return __builtin_nontemporal_load(p); }
__device__ __forceinline__ f32x2_t ld_x(gptr<f32x2_t> p) { return __builtin_nontemporal_load(p); }
__device__ __forceinline__ f32x4 ld_x(gptr<f32x4> p) { return __builtin_nontemporal_load(p); }
// device-coherent accesses (data crossing XCDs)
__device__ __forceinline__ float ld_dev(const float* p) {
  return __hip_atomic_load((float*)p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float ld_dev(gptr<float> p) {
  return __hip_atomic_load((gw<float>)p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ unsigned ld_flag(const unsigned* p) {
  return __hip_atomic_load((unsigned*)p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ bool tag_reached(unsigned v, unsigned tag) { return (int)(v - tag) >= 0; }

// ------------------------------------------------------------------ waits and signals

struct Wg {
  int x, r, g;       // XCD, rank, x * 32 + r
  unsigned E;        // this pass's number
  unsigned tagbase;  // E * tags per pass
  int* sh;           // LDS words shared by the workgroup
  unsigned char* lds;  // the workgroup's dynamic LDS
  const int* plan;   // this workgroup's plan row, copied to LDS
  const unsigned long long* lwt;  // the per-layer parameter pointers, copied to LDS
};

// the dependency of a stage: flags of stage id on XCD wx (-1: all XCDs) at
// tag; on = false when there is none.  Stages load what does not depend on
// it (weights, cached K/V) before they wait.
struct WaitSpec {
  int id, wx;
  unsigned tag;
  bool on;
  int sl, sfid;  // layer and flag id of the caller's stage timestamps
};

__device__ __forceinline__ unsigned tag_of(const Wg& w, int l, int s) {
  return w.tagbase + (unsigned)(l * kFStages + s) + 1u;
}

__device__ __forceinline__ void raise_abort(const FusedArgs& a, unsigned code) {
  if (__hip_atomic_exchange(&a.ctl[FZ_ABORT], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == 0u) {
    __hip_atomic_store(&a.ctl[FZ_WHY], code, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (a.err) __hip_atomic_fetch_add(a.err, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

// Workgroup barrier that orders LDS accesses only: outstanding global stores
// are not waited for (signal() waits for them before a stage is published).
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// Barrier of waves 0..3 alone (the other four keep their own loads going):
// a counter in LDS that every round raises by 4; a wave leaves when the
// round it joined is complete.  LDS accesses of a wave are performed in
// order, so its writes before the barrier are visible after it.
constexpr int QW = 4;  // waves that run the pre-stage rows
__device__ __forceinline__ void q_barrier(const Wg& w) {
  __attribute__((address_space(3))) unsigned* cnt = (__attribute__((address_space(3))) unsigned*)(w.sh + 4);
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  unsigned old = 0;
  if ((threadIdx.x & 63) == 0) old = __hip_atomic_fetch_add(cnt, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
  old = __builtin_amdgcn_readfirstlane(old);
  const unsigned target = (old / QW + 1) * QW;
  while ((int)(__hip_atomic_load(cnt, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP) - target) < 0)
    __builtin_amdgcn_s_sleep(1);
}

// Wave 0 alone polls until the flags of stage s reach tag: the 32 of XCD xs,
// or all 256 when xs < 0.  No workgroup barrier: the other waves go on with
// their own work.  Returns false (in every lane) on abort or timeout.  On
// success the CU's L1 lines are dropped before the wave's own later loads
// (acquire: a wave's memory operations reach the cache in order, and the
// flags' values were consumed, so they are complete).  The workgroup-scope
// invalidate drops the L1 only; the agent-scope one would also drop the
// XCD's L2.
__device__ __forceinline__ bool poll_w0(const FusedArgs& a, const Wg& w, int s, int xs, unsigned tag) {
  const int lane = threadIdx.x & 63;
  const unsigned* f = a.flags + (size_t)s * kFGroups;
  const unsigned long long t0 = now();
  bool ok = false;
  for (;;) {
    bool mine;
    if (xs < 0) {
      const unsigned v0 = ld_flag(f + 4 * lane), v1 = ld_flag(f + 4 * lane + 1);
      const unsigned v2 = ld_flag(f + 4 * lane + 2), v3 = ld_flag(f + 4 * lane + 3);
      mine = tag_reached(v0, tag) && tag_reached(v1, tag) && tag_reached(v2, tag) && tag_reached(v3, tag);
    } else {
      mine = lane >= kFRanks || tag_reached(ld_flag(f + xs * kFRanks + lane), tag);
    }
    if (__all(mine)) {
      ok = true;
      break;
    }
    if (ld_flag(&a.ctl[FZ_ABORT])) break;
    if (now() - t0 > a.timeout) {
      if (lane == 0) raise_abort(a, 0x100u + (unsigned)s);
      break;
    }
    __builtin_amdgcn_s_sleep(1);
  }
  if (ok) asm volatile("buffer_inv sc0" ::: "memory");
  return ok;
}

// The same wait for the whole workgroup: wave 0 polls, the others wait at an
// LDS-only barrier (loads they issued before it, weights or cached K/V, stay
// in flight), then each wave drops the L1 before its own loads.
__device__ __forceinline__ bool wait_flags(const FusedArgs& a, const Wg& w, int s, int xs, unsigned tag) {
  if (threadIdx.x < 64) {
    const bool ok = poll_w0(a, w, s, xs, tag);
    if (threadIdx.x == 0) w.sh[0] = ok;
  }
  lds_barrier();
  const bool ok = w.sh[0] != 0;
  lds_barrier();
  if (threadIdx.x >= 64) asm volatile("buffer_inv sc0" ::: "memory");
  return ok;
}

// Publishes stage s of layer l: every thread's stores complete, then one flag.
__device__ __forceinline__ void signal(const FusedArgs& a, const Wg& w, int l, int s, bool cross_xcd) {
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  if (threadIdx.x == 0) {
    unsigned* f = a.flags + (size_t)s * kFGroups + w.g;
    if (cross_xcd) __hip_atomic_store(f, tag_of(w, l, s), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    else __hip_atomic_store(f, tag_of(w, l, s), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
  }
}

// Publishes stage s of layer l for work wave 0 did alone (its LayerNorm rows
// or attention merges, read inside the XCD): its stores complete, then the
// flag.
__device__ __forceinline__ void signal_w0(const FusedArgs& a, const Wg& w, int l, int s) {
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  if (threadIdx.x == 0)
    __hip_atomic_store(a.flags + (size_t)s * kFGroups + w.g, tag_of(w, l, s), __ATOMIC_RELAXED,
                       __HIP_MEMORY_SCOPE_WORKGROUP);
}

// stage timestamps (when the session traces): entry, dependency met, done
__device__ __forceinline__ void stamp(const FusedArgs& a, const Wg& w, int l, int s, int k) {
  if (a.trace && threadIdx.x == 0)
    a.trace[(((size_t)w.g * (a.L + 1) + l) * kFStages + s) * 3 + k] = now();
}

// ------------------------------------------------------------------ per-layer parameters

enum LwSlot { LW_QKV = 0, LW_O, LW_FC, LW_PR, LB_QKV, LB_O, LB_FC, LB_PR, LN1G, LN1B, LN2G, LN2B };


// (read from the workgroup's LDS copy: an LDS read never holds up the wave's
// flag polls, which a global load issued before them would)
__device__ __forceinline__ const void* lw(const Wg& w, int l, int slot) {
  return (const void*)((const __attribute__((address_space(3))) unsigned long long*)w.lwt)[l * kLwSlots + slot];
}

// ------------------------------------------------------------------ LayerNorm of one node row
//
// mode 0: x = wte[token] + wpe[position] (first layer);
// mode 1: x += float((S + bias) * 2^-32), S the fixed-point sum of every
//         XCD's partial of the residual GEMM (device-coherent loads), the
//         bias rounded to the same units: one rounding per element;
// then a = (x - mean) / sqrt(var + eps) * g + b into this XCD's GEMM input.
// The sums of sub-layer k live in buffer k % 3 (see xs_zero).
// One wave: lane i takes the float4 chunks i, i + 64, ... (C per lane, so
// d <= 256 C); sums run over the lane's chunks in order, then across lanes
// by butterfly.  The other waves of the workgroup are free meanwhile.

// Sum over the 64 lanes of a wave, the same value in every lane, in a fixed
// order: DPP exchanges inside each row of 16 lanes (xor 1, xor 2, half-row
// mirror, row mirror), then the four row sums in lane order.
template <int CTRL>
__device__ __forceinline__ float dpp_f(float x) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), CTRL, 0xf, 0xf, false));
}
__device__ __forceinline__ float wave_sum(float x) {
  x += dpp_f<0xB1>(x);   // quad_perm [1,0,3,2]
  x += dpp_f<0x4E>(x);   // quad_perm [2,3,0,1]
  x += dpp_f<0x141>(x);  // row_half_mirror
  x += dpp_f<0x140>(x);  // row_mirror
  const float r0 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 0));
  const float r1 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 16));
  const float r2 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 32));
  const float r3 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 48));
  return (r0 + r1) + (r2 + r3);
}

// Max / sum over each half-wave (lanes 0..31, 32..63), the half's value in
// each of its lanes: DPP inside rows of 16, then the half's two row values
// in lane order.
__device__ __forceinline__ float half_pick(float x, float (*op)(float, float)) {
  const float r0 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 0));
  const float r1 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 16));
  const float r2 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 32));
  const float r3 = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), 48));
  return (threadIdx.x & 32) ? op(r2, r3) : op(r0, r1);
}
__device__ __forceinline__ float fmax_f(float a, float b) { return fmaxf(a, b); }
__device__ __forceinline__ float fadd_f(float a, float b) { return a + b; }
__device__ __forceinline__ float half_max(float x) {
  x = fmaxf(x, dpp_f<0xB1>(x));
  x = fmaxf(x, dpp_f<0x4E>(x));
  x = fmaxf(x, dpp_f<0x141>(x));
  x = fmaxf(x, dpp_f<0x140>(x));
  return half_pick(x, fmax_f);
}
__device__ __forceinline__ float half_sum(float x) {
  x += dpp_f<0xB1>(x);
  x += dpp_f<0x4E>(x);
  x += dpp_f<0x141>(x);
  x += dpp_f<0x140>(x);
  return half_pick(x, fadd_f);
}

// Fixed-point residual sums.  Sub-layer k (2l: out-projection of layer l,
// 2l + 1: its down-projection) is summed in buffer k % 3 of xacc.  A buffer
// is cleared (each XCD its eighth of the columns of the rows below N) by the
// LayerNorm that consumes the sum after it: the LayerNorm of sub-layer k
// clears buffer (k - 1) % 3, which every XCD has read by then (that
// LayerNorm waits for every XCD's sub-layer k, which each XCD runs after
// its own LayerNorm of k - 1), and which is next added to by sub-layer
// k + 2, which every XCD runs after the LayerNorm of k + 1, itself waiting
// for every XCD's sub-layer k + 1 and so for every XCD's clearing.  The
// first layer's LayerNorm clears buffers 0 and 1, and the first QKV stage
// waits for all 256 workgroups' first LayerNorm, so a pass starts from clear
// sums whatever the pass before it left (one that ended early included).
constexpr double kFixScale = 4294967296.0;     // 2^32 units per 1.0
constexpr float kFixMax = 134217728.f;         // 2^27: nine terms stay below 2^63
__device__ __forceinline__ gw<long long> xs_row(const FusedArgs& a, int k, int n) {
  return (gw<long long>)a.xacc + ((size_t)(k % 3) * kFMaxN + n) * a.d;
}
// this XCD's eighth of the columns of row n of buffer b, stored as zeros
// (device-coherent stores, as the atomics that follow are performed beyond
// the XCD's L2); run by waves 0..3
__device__ __forceinline__ void xs_zero(const FusedArgs& a, const Wg& w, int b, int n) {
  const int c8 = a.d / kFXcd, tid = opq_tid();
  for (int c = tid; c < c8; c += QW * 64)
    __hip_atomic_store(xs_row(a, b, n) + w.x * c8 + c, 0ll, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// adds this XCD's partial v of output o of node n to sub-layer k's sum; a
// magnitude past 2^27 (or NaN) is counted in err (one count per wave) and
// clamped, so the nine terms of a sum cannot overflow
__device__ __forceinline__ void xs_add(const FusedArgs& a, int k, int n, int o, float v) {
  const bool over = !(fabsf(v) <= kFixMax);
  const unsigned long long m = __builtin_amdgcn_ballot_w64(over);
  if (m && (int)__builtin_amdgcn_mbcnt_hi(~0u, __builtin_amdgcn_mbcnt_lo(~0u, 0u)) == __builtin_ctzll(m))
    __hip_atomic_fetch_add(a.err, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  const float vc = over ? (v > 0.f ? kFixMax : -kFixMax) : v;
  __hip_atomic_fetch_add(xs_row(a, k, n) + o, (long long)llrint((double)vc * kFixScale), __ATOMIC_RELAXED,
                         __HIP_MEMORY_SCOPE_AGENT);
}

// Waves 0..3 (256 threads) normalise R node rows n0, n0 + 32, ... (those
// below N) together: thread t takes the float4 chunks t, t + 256, ... of
// each row (C per thread, d <= 1024 C); sums run over the thread's chunks in
// order, across its wave by DPP, then over the four waves in wave order.
// Wave 0 polls with nothing else in flight (a wave's loads complete in
// order, so anything issued before would delay the poll); every load of
// every row is issued together right after it.
template <int C, int R, bool RE>
__device__ __forceinline__ bool ln_rows_q(const FusedArgs& a, const Wg& w, const WaitSpec& ws, int n0, int mode,
                                          gptr<uint16_t> bias, int kin, unsigned zmask, gptr<uint16_t> g,
                                          gptr<uint16_t> b, uint16_t* act) {
  const int d = a.d, nc = d / 4, tid = opq_tid(), wv = tid >> 6;
  float* red = (float*)(w.sh + 16);  // [R][8]
  if (mode != 0 && ws.on) {
    if (wv == 0) {
      const bool ok = poll_w0(a, w, ws.id, ws.wx, ws.tag);
      if (tid == 0) w.sh[5] = ok;
    }
    q_barrier(w);
    if (w.sh[5] == 0) return false;
    if (wv > 0) asm volatile("buffer_inv sc0" ::: "memory");
    stamp(a, w, ws.sl, ws.sfid, 1);
  }
  int nr[R];
#pragma unroll
  for (int j = 0; j < R; ++j) nr[j] = min(n0 + j * kFRanks, a.N - 1);  // (rows past N repeat the last; not stored)
  const gptr<u32x2> g4 = (gptr<u32x2>)opq(g), b4 = (gptr<u32x2>)opq(b);
  const gw<uint16_t> actg = opq(act);
  int cc[C];
#pragma unroll
  for (int i = 0; i < C; ++i) cc[i] = min(tid + QW * 64 * i, nc - 1);
  auto bf4 = [](u32x2 u) {
    return (f32x4){__uint_as_float(u.x << 16), __uint_as_float(u.x & 0xffff0000u), __uint_as_float(u.y << 16),
                   __uint_as_float(u.y & 0xffff0000u)};
  };
  f32x4 v[R][C];
  u32x2 gr[C], br[C];
#pragma unroll
  for (int i = 0; i < C; ++i) {
    gr[i] = g4[cc[i]];
    br[i] = b4[cc[i]];
  }
  if (RE && mode == 0) {
    // the pass starts at a later layer: the rows' residual stream as given
#pragma unroll
    for (int j = 0; j < R; ++j) {
      const gptr<f32x4> xi = (gptr<f32x4>)opq(a.x_in + (size_t)nr[j] * d);
#pragma unroll
      for (int i = 0; i < C; ++i) v[j][i] = xi[cc[i]];
    }
  } else if (mode == 0) {
    u32x2 tr[R][C], pr[R][C];
#pragma unroll
    for (int j = 0; j < R; ++j) {
      const int tok = ld_x(a.tree + nr[j]), pos = ld_x(a.tree + a.max_nodes + nr[j]);
      const gptr<u32x2> te = (gptr<u32x2>)(opq(a.wte) + (size_t)tok * d);
      const gptr<u32x2> pe = (gptr<u32x2>)(opq(a.wpe) + (size_t)pos * d);
#pragma unroll
      for (int i = 0; i < C; ++i) {
        tr[j][i] = te[cc[i]];
        pr[j][i] = pe[cc[i]];
      }
    }
#pragma unroll
    for (int j = 0; j < R; ++j)
#pragma unroll
      for (int i = 0; i < C; ++i) v[j][i] = bf4(tr[j][i]) + bf4(pr[j][i]);
  } else {
    // the rows' fixed-point sums: device-coherent 16-byte loads (two per
    // float4 chunk)
    const __amdgpu_buffer_rsrc_t srs = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(a.xacc + (size_t)(kin % 3) * kFMaxN * d), (short)0, (int)(kFMaxN * d * 8), 0x00020000);
    u32x4 sv[R][C][2];
#pragma unroll
    for (int j = 0; j < R; ++j)
#pragma unroll
      for (int i = 0; i < C; ++i)
#pragma unroll
        for (int hf = 0; hf < 2; ++hf)
          sv[j][i][hf] = __builtin_bit_cast(
              u32x4, __builtin_amdgcn_raw_buffer_load_b128(srs, (unsigned)(32 * cc[i] + 16 * hf),
                                                           (unsigned)((size_t)nr[j] * d * 8), CP_SC1));
    const gptr<u32x2> c4 = (gptr<u32x2>)opq(bias);
    f32x4 xv[R][C];
    u32x2 cr[C];
#pragma unroll
    for (int i = 0; i < C; ++i) cr[i] = c4[cc[i]];
#pragma unroll
    for (int j = 0; j < R; ++j) {
      const gptr<f32x4> xr = (gptr<f32x4>)opq(a.xr + ((size_t)w.x * kFMaxN + nr[j]) * d);
#pragma unroll
      for (int i = 0; i < C; ++i) xv[j][i] = xr[cc[i]];
    }
    // the sum plus the bias in the same units, rounded once to float
    auto fx = [](unsigned lo, unsigned hi, float bv) {
      const long long s = (long long)(((unsigned long long)hi << 32) | lo) + (long long)llrint((double)bv * kFixScale);
      return (float)((double)s * (1.0 / kFixScale));
    };
#pragma unroll
    for (int j = 0; j < R; ++j)
#pragma unroll
      for (int i = 0; i < C; ++i) {
        const f32x4 bb = bf4(cr[i]);
        const f32x4 acc = {fx(sv[j][i][0].x, sv[j][i][0].y, bb[0]), fx(sv[j][i][0].z, sv[j][i][0].w, bb[1]),
                           fx(sv[j][i][1].x, sv[j][i][1].y, bb[2]), fx(sv[j][i][1].z, sv[j][i][1].w, bb[3])};
        v[j][i] = xv[j][i] + acc;
      }
  }
  // clear the buffers this stage is due to clear (its rows, this XCD's
  // columns); issued after every load above
#pragma unroll
  for (int zb = 0; zb < 3; ++zb)
    if (zmask >> zb & 1u)
#pragma unroll
      for (int j = 0; j < R; ++j)
        if (n0 + j * kFRanks < a.N) xs_zero(a, w, zb, n0 + j * kFRanks);
  float sm[R];
#pragma unroll
  for (int j = 0; j < R; ++j) {
    const gw<f32x4> xr = (gw<f32x4>)opq(a.xr + ((size_t)w.x * kFMaxN + nr[j]) * d);
    float sj = 0.f;
#pragma unroll
    for (int i = 0; i < C; ++i) {
      if (tid + QW * 64 * i < nc) {
        if (n0 + j * kFRanks < a.N) xr[tid + QW * 64 * i] = v[j][i];
        sj += ((v[j][i][0] + v[j][i][1]) + (v[j][i][2] + v[j][i][3]));
      }
    }
    sm[j] = wave_sum(sj);
    if ((tid & 63) == 0) red[8 * j + wv] = sm[j];
  }
  q_barrier(w);
  float mean[R], qs[R];
#pragma unroll
  for (int j = 0; j < R; ++j) {
    mean[j] = ((red[8 * j] + red[8 * j + 1]) + (red[8 * j + 2] + red[8 * j + 3])) / d;
    float q = 0.f;
#pragma unroll
    for (int i = 0; i < C; ++i) {
      if (tid + QW * 64 * i < nc) {
        const f32x4 c = v[j][i] - mean[j];
        q += ((c[0] * c[0] + c[1] * c[1]) + (c[2] * c[2] + c[3] * c[3]));
      }
    }
    qs[j] = wave_sum(q);
    if ((tid & 63) == 0) red[8 * j + 4 + wv] = qs[j];
  }
  q_barrier(w);
#pragma unroll
  for (int j = 0; j < R; ++j) {
    if (n0 + j * kFRanks >= a.N) break;
    const float rden =
        1.0f / sqrtf(((red[8 * j + 4] + red[8 * j + 5]) + (red[8 * j + 6] + red[8 * j + 7])) / d + a.eps);
#pragma unroll
    for (int i = 0; i < C; ++i) {
      const int c = tid + QW * 64 * i;
      if (c < nc) {
        const f32x4 gv = bf4(gr[i]), bv = bf4(br[i]);
        const f32x4 y = (v[j][i] - mean[j]) * rden * gv + bv;
        st_act4(actg, nr[j], 4 * c, d / 32, y[0], y[1], y[2], y[3], a.err);
      }
    }
  }
  return true;
}

// ------------------------------------------------------------------ attention merge and pre-stages
//
// An attention unit leaves one record per node of its tile: max, sum, -, -,
// output[64].
constexpr int AREC = DH + 4;                // part record: max, sum, -, -, output

__device__ __forceinline__ gw<float> part_rec(const FusedArgs& a, int h, int t, int u, int nl) {
  return (gw<float>)a.apart + ((((size_t)h * 4 + t) * (a.att_units + 1) + u) * 16 + nl) * AREC;
}

// The whole workgroup merges the parts of (head h, tile t) in part order:
// thread i takes dims 2 (i % 32), +1 of node i / 32.  Per (node, dim) the
// arithmetic is the online-softmax merge of the parts, in order.
__device__ __forceinline__ void merge_tile(const FusedArgs& a, int h, int t) {
  const int tid = opq_tid(), nl = tid >> 5, d0 = 2 * (tid & 31), S = a.att_units;
  float M = -INFINITY, Ls = 0.f, O0 = 0.f, O1 = 0.f;
  constexpr int MJ = 4;  // parts loaded per round trip
  for (int j0 = 0; j0 <= S; j0 += MJ) {
    f32x2_t ml[MJ], ov[MJ];
#pragma unroll
    for (int jj = 0; jj < MJ; ++jj) {
      const gptr<float> rec = (gptr<float>)part_rec(a, h, t, min(j0 + jj, S), nl);
      ml[jj] = ld_x((gptr<f32x2_t>)rec);
      ov[jj] = ld_x((gptr<f32x2_t>)(rec + 4 + d0));
    }
#pragma unroll
    for (int jj = 0; jj < MJ; ++jj) {
      if (j0 + jj > S) break;
      const float mj = ml[jj][0], lj = ml[jj][1];
      if (mj == -INFINITY) continue;
      const float mn = fmaxf(M, mj);
      const float al = __expf(M - mn), wj = __expf(mj - mn);
      Ls = fmaf(Ls, al, lj * wj);
      O0 = fmaf(O0, al, ov[jj][0] * wj);
      O1 = fmaf(O1, al, ov[jj][1] * wj);
      M = mn;
    }
  }
  const int n = 16 * t + nl;
  if (n < a.N) {
    const gw<uint16_t> fo = opq(a.fo);
    st_act(fo, n, h * DH + d0, a.d / 32, O0 / Ls, a.err);
    st_act(fo, n, h * DH + d0 + 1, a.d / 32, O1 / Ls, a.err);
  }
}

// After a unit of (head h, tile t) stored its part: once every wave's part
// stores are complete, one lane counts the unit in the tile's counter with an
// atomic increment that wraps after the tile's last unit (S prefix units +
// the root unit); the unit that reads the count S (the last one to arrive)
// merges the tile.  The increments of a tile are serialised at the counter,
// so exactly one unit merges, after every part is stored, and the counter is
// back at 0 for the next layer.  (A flag per unit, each unit reading all its
// tile's flags after storing its own, let the two last units miss each
// other's flags now and then, so that no unit merged: on this hardware a
// completed store is not yet seen by another CU's load for a short time.)
__device__ __forceinline__ void unit_done(const FusedArgs& a, const Wg& w, int l, int h, int t, int j) {
  (void)l;
  (void)j;
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  lds_barrier();
  if (threadIdx.x == 0) {
    const unsigned old = __builtin_amdgcn_atomic_inc32(a.tile_ctr + (size_t)h * 4 + t, (unsigned)a.att_units,
                                                       __ATOMIC_RELAXED, "agent");
    w.sh[6] = old == (unsigned)a.att_units;
  }
  lds_barrier();
  const bool last = w.sh[6] != 0;
  lds_barrier();
  if (last) {
    asm volatile("buffer_inv sc0" ::: "memory");
    merge_tile(a, h, t);
  }
}

// What waves 0..3 do before a weight GEMM while the other waves' weight loads
// are in flight: a LayerNorm stage's rows; then they publish that stage.
struct PreSpec {
  int kind;  // 0 nothing, 1 LayerNorm rows
  int l, fid;
  WaitSpec ws;
  int mode;
  gptr<uint16_t> bias, g, b;
  int kin;          // the sub-layer whose fixed-point sums the rows add (mode 1)
  unsigned zmask;   // sum buffers this stage clears (bit b: buffer b)
  uint16_t* act;
  // after the rows, waves 1..3 copy these weight fragments (row blocks
  // wrbs[0 .. wn) of W, k-steps [wk0, wk1) of KC) into LDS at wdst, in
  // (row block, k-step) order, for a GEMM two stages on (wn = 0: none)
  int wn, wk0, wk1, wKC, wdst;  // (wdst: byte offset in LDS)
  const int* wrbs;
  gptr<u32x4> wW;
};

constexpr int WST = 16 * 1024;                              // LDS offset of the down-projection's staged weights
constexpr int WST_FRAGS = (73728 + 34816 + 4096 - WST) / 1024;  // 1 KB fragments that fit below sh
constexpr int WO_FRAGS = 24;  // the out-projection's staged fragments, above the parameter table

// Every weight fragment is read by exactly one workgroup of the pass, once,
// so weights are loaded non-temporal (the nt cache-policy bit; for the
// register loads __builtin_nontemporal_load): streaming about 4.9 MB through
// each XCD's 4 MB L2 per layer would otherwise evict the residual copies,
// activations and attention parts the next stages read back.
constexpr int kWeightCpol = 2;

// Copies weight fragments f = wv - 1, wv - 1 + nw, ... < n * nk (row block
// rbs[f / nk] (an LDS list), k-step k0 + f % nk of a matrix of KC k-steps)
// into LDS at dst + f * fragment bytes, by waves 1.. of a stage (nw of them).
// float16 fragments (1 KB) take one 16-byte copy per lane; 8-bit fragments
// (512 B) go two at a time (see below), so the LDS image equals the
// fragments either way.
template <bool Q8>
__device__ __forceinline__ void stage_frags(gptr<u32x4> W, const int* rbs, int n, int k0, int nk, int KC,
                                            unsigned char* dst, int wv, int nw) {
  const int lane = threadIdx.x & 63, tot = n * nk;
  if constexpr (!Q8) {
    const gptr<u32x4> Wv = opq(W) + lane;
    for (int f = wv - 1; f < tot; f += nw) {
      const int r = f / nk, k = k0 + f - r * nk;
      const int rb = ((const __attribute__((address_space(3))) int*)rbs)[r];
      __builtin_amdgcn_global_load_lds((const void*)(Wv + ((size_t)rb * KC + k) * 64),
                                       (lds_void*)(dst + (size_t)f * 1024), 16, 0, kWeightCpol);
    }
  } else {
    // two consecutive k-steps of a row block are 1 KB contiguous in memory
    // and in LDS: one 16-byte copy per lane; an odd last k-step of a row
    // block goes as two 4-byte copies
    const int np = nk >> 1, per = np + (nk & 1);
    const gptr<u32x4> W16 = opq(W) + lane;
    const gptr<unsigned> W4 = (gptr<unsigned>)opq(W) + lane;
    (void)tot;
    for (int c = wv - 1; c < n * per; c += nw) {
      const int r = c / per, j = c - r * per, k = k0 + 2 * j;
      const int rb = ((const __attribute__((address_space(3))) int*)rbs)[r];
      unsigned char* d = dst + (size_t)(r * nk + 2 * j) * 512;
      if (j < np) {
        __builtin_amdgcn_global_load_lds((const void*)(W16 + ((size_t)rb * KC + k) * 32), (lds_void*)d, 16, 0,
                                         kWeightCpol);
      } else {
        const gptr<unsigned> src = W4 + ((size_t)rb * KC + k) * 128;
        __builtin_amdgcn_global_load_lds((const void*)src, (lds_void*)d, 4, 0, kWeightCpol);
        __builtin_amdgcn_global_load_lds((const void*)(src + 64), (lds_void*)(d + 256), 4, 0, kWeightCpol);
      }
    }
  }
}

// Run by waves 0..3 together: the LayerNorm rows, then the stage is
// published (the four waves' stores complete, then wave 0 writes the flag).
template <bool Q8, bool RE>
__device__ __forceinline__ bool do_pre(const FusedArgs& a, const Wg& w, const PreSpec& ps) {
  if (ps.kind == 0) return true;
  bool ok = true;
  if (ps.kind == 1 && w.r < a.N) {
    // this rank's rows: w.r and (at more than 32 nodes) w.r + 32, together
    const bool two = w.r + kFRanks < a.N;
    if (a.d <= 1024)
      ok = two ? ln_rows_q<1, 2, RE>(a, w, ps.ws, w.r, ps.mode, ps.bias, ps.kin, ps.zmask, ps.g, ps.b, ps.act)
               : ln_rows_q<1, 1, RE>(a, w, ps.ws, w.r, ps.mode, ps.bias, ps.kin, ps.zmask, ps.g, ps.b, ps.act);
    else
      ok = two ? ln_rows_q<2, 2, RE>(a, w, ps.ws, w.r, ps.mode, ps.bias, ps.kin, ps.zmask, ps.g, ps.b, ps.act)
               : ln_rows_q<2, 1, RE>(a, w, ps.ws, w.r, ps.mode, ps.bias, ps.kin, ps.zmask, ps.g, ps.b, ps.act);
  }
  if (!ok) return false;
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  q_barrier(w);
  if (threadIdx.x == 0) {
    // (the first layer's LayerNorm is waited for by every XCD: a
    // device-coherent flag; the others are read inside the XCD)
    unsigned* f = a.flags + (size_t)ps.fid * kFGroups + w.g;
    if (ps.mode == 0) __hip_atomic_store(f, tag_of(w, ps.l, ps.fid), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    else __hip_atomic_store(f, tag_of(w, ps.l, ps.fid), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
  }
  stamp(a, w, ps.l, ps.fid, 2);
  if (ps.wn > 0 && threadIdx.x >= 64) {
    // (not wave 0: its polls must not wait behind these loads; the stage's
    // closing vmcnt(0) and barrier complete them before the GEMM reads them)
    stage_frags<Q8>(ps.wW, ps.wrbs, ps.wn, ps.wk0, ps.wk1 - ps.wk0, ps.wKC, w.lds + ps.wdst, threadIdx.x >> 6,
                    QW - 1);
  }
  return true;
}

// ------------------------------------------------------------------ skinny GEMM of one task
//
// Y[n][o] = sum_k A[n][k] W[o][k] for the task's row blocks (up to RBM, any
// order) over k-steps [kc0, kc1).  Wave w takes k-steps kc0 + w, kc0 + w + 4,
// ..., U steps of loads in flight; per step it multiplies every row block's
// weight fragment into every 16-node activation fragment on
// v_mfma_f32_16x16x32_f16.  The four waves are summed in wave order through
// LDS, one row block at a time, and the epilogue writes each output.

enum FEpi { FE_QKV = 0, FE_WO, FE_FC, FE_WPR, FE_HEAD };

__device__ __forceinline__ void epilogue(const FusedArgs& a, const Wg& w, int epi, int l, int n, int o, float v) {
  const int d = a.d;
  switch (epi) {
    case FE_QKV:
      if (o < d) {
        a.q[(size_t)n * d + o] = v;
      } else {
        const int oo = o < 2 * d ? o - d : o - 2 * d;
        const int h = oo / DH, e = oo - h * DH;
        uint16_t* dst = o < 2 * d ? a.kt : a.vt;
        dst[(((size_t)l * a.H + h) * a.max_nodes + n) * DH + e] = f2bf(v);
      }
      break;
    case FE_WO: xs_add(a, 2 * l, n, o, v); break;
    case FE_FC: st_act(opq(a.ff), n, o, a.M / 32, gelu_tanh(v), a.err); break;
    case FE_WPR: xs_add(a, 2 * l + 1, n, o, v); break;
    default: a.logits[(size_t)n * a.V + o] = v; break;
  }
}

// The LM head's running maximum per node of this workgroup (greedy accept
// without re-reading the logits): thread t owns epilogue slots t and t + 512,
// i.e. row (t % 16) of node t / 16 and of node t / 16 + 32, in every row
// block; a slot keeps its largest logit and, among equals, the lowest token.
struct HeadBest {
  float v[2];
  int o[2];
};

// One GEMM task of RB row blocks: rbs[0 .. nrb) (plan entries) or, with rbs
// null, nrb consecutive ones from rb_first; row blocks past nrb repeat the
// last one and are not stored.  Q8: the matrix is in 8-bit fragments (512 B,
// widened to float16 in registers) followed by its rows' float32 scales
// ([ceil(M / 16) 16]); each output is scaled by its row's before the bias.
template <int NT, int RB, int U, bool Q8, bool RE>
__device__ __forceinline__ bool gemm_rb(const FusedArgs& a, const Wg& w, const WaitSpec& ws, int epi, int l,
                                        const int* rbs, int rb_first, int nrb, gptr<uint16_t> bias, gptr<u32x4> Wp,
                                        int KC, int M, int kc0, int kc1, const uint16_t* act, int act_kc,
                                        float* red, const PreSpec& ps, int wofs, HeadBest& hb, bool track) {
  constexpr int NN = 16 * NT, NCW = NWV - QW;
  using WT = typename std::conditional<Q8, u32x2, u32x4>::type;
  // Waves 4..7 compute: wave 4 + c takes k-steps kc0 + c, kc0 + c + 4, ...,
  // and loads their weights first thing.  Waves 0..3 run the pre-stage
  // meanwhile; then wave 0, with nothing in flight, waits for this stage's
  // dependency.  The wave index and step count are scalars, so the step
  // guards below are scalar branches: an MFMA ignores EXEC and must never
  // sit under a lane mask.
  const int tid = opq_tid(), wv = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
  const int cw = wv - QW;
  const int nsteps = wv >= QW && kc1 - kc0 > cw ? (kc1 - kc0 - cw + NCW - 1) / NCW : 0;
  Wp = opq(Wp);
  const gptr<WT> Wq = (gptr<WT>)Wp;
  const gptr<uint16_t> actg = opq(act);
  bias = opq(bias);
  int rbv[RB];
#pragma unroll
  for (int r = 0; r < RB; ++r) {
    const int rr = min(r, nrb - 1);
    rbv[r] = rbs ? ((const __attribute__((address_space(3))) int*)rbs)[rr] : rb_first + rr;  // (LDS copy)
  }
  // this thread's epilogue row of every row block is tid % 16: its bias is
  // loaded before the k-loop
  // The load is unconditional (a GEMM without bias reads a word of its own
  // weights instead, and discards it in the epilogue): a conditional load
  // would be waited for on the spot.
  const bool has_bias = bias != nullptr;
  const gptr<uint16_t> bsrc = has_bias ? bias : (gptr<uint16_t>)Wp;
  uint16_t bias_r[RB];
  float scale_r[RB];
  gptr<WT> wb[RB];
#pragma unroll
  for (int r = 0; r < RB; ++r) wb[r] = Wq + (size_t)rbv[r] * KC * 64 + lane;
  const gptr<u32x4> ab = (gptr<u32x4>)actg + lane;
  WT wq[U][RB];
  u32x4 bq[U][NT];
  const int klast = kc1 - 1;
  const int nk = kc1 - kc0;
  const __attribute__((address_space(3))) WT* wl =
      (const __attribute__((address_space(3))) WT*)((unsigned char*)red + wofs) + lane;
  auto load_w = [&](int s, int u) {
    const int kc = min(kc0 + cw + NCW * s, klast);
    if (wofs) {
      // staged in LDS by the stage before the last ((row block, k-step) order)
#pragma unroll
      for (int r = 0; r < RB; ++r) wq[u][r] = wl[(min(r, nrb - 1) * nk + (kc - kc0)) * 64];
    } else {
      // (non-temporal: see kWeightCpol)
#pragma unroll
      for (int r = 0; r < RB; ++r) wq[u][r] = __builtin_nontemporal_load(&wb[r][(size_t)kc * 64]);
    }
  };
  auto load_a = [&](int s, int u) {
    const int kc = min(kc0 + cw + NCW * s, klast);
#pragma unroll
    for (int t = 0; t < NT; ++t) bq[u][t] = ld_x(ab + ((size_t)t * act_kc + kc) * 64);
  };
  auto load_step = [&](int s, int u) {
    load_w(s, u);
    load_a(s, u);
  };
  f32x4 acc[RB][NT];
#pragma unroll
  for (int r = 0; r < RB; ++r)
#pragma unroll
    for (int t = 0; t < NT; ++t) acc[r][t] = (f32x4){0.f, 0.f, 0.f, 0.f};
  // the first U steps' weights do not depend on the previous stage: they are
  // in flight while the workgroup waits for it
  // only the steps this wave owns are loaded (the step bounds are uniform
  // per wave, so the guards are scalar branches)
  // (the loads sit in the branch wave 0 does not take, so the weight
  // registers are not live across the pre-stage's code)
  if (wv < QW) {
    bool ok = do_pre<Q8, RE>(a, w, ps);
    if (wv == 0) {
      stamp(a, w, ws.sl, ws.sfid, 0);
      if (ok && ws.on) ok = poll_w0(a, w, ws.id, ws.wx, ws.tag);
      if (lane == 0) w.sh[0] = ok;
    }
  } else {
#pragma unroll
    for (int u = 0; u < U; ++u)
      if (u < nsteps) load_w(u, u);
  }
  lds_barrier();
  if (w.sh[0] == 0) return false;
  lds_barrier();
  if (wv > 0) asm volatile("buffer_inv sc0" ::: "memory");
  stamp(a, w, ws.sl, ws.sfid, 1);
  // the bias is loaded only now, so that nothing sits ahead of wave 0's polls
#pragma unroll
  for (int r = 0; r < RB; ++r) bias_r[r] = bsrc[rbv[r] * 16 + (tid & 15)];
  if constexpr (Q8) {
    const gptr<float> sc = (gptr<float>)(Wq + (size_t)((M + 15) / 16) * KC * 64);
#pragma unroll
    for (int r = 0; r < RB; ++r) scale_r[r] = sc[rbv[r] * 16 + (tid & 15)];
  }
#pragma unroll
  for (int u = 0; u < U; ++u)
    if (u < nsteps) load_a(u, u);
  __builtin_amdgcn_sched_barrier(0);
  for (int s0 = 0; s0 < nsteps; s0 += U) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      if (s0 + u < nsteps) {
#pragma unroll
        for (int r = 0; r < RB; ++r)
#pragma unroll
          for (int t = 0; t < NT; ++t)
            acc[r][t] = __builtin_amdgcn_mfma_f32_16x16x32_f16(wfrag(wq[u][r]), __builtin_bit_cast(f16x8, bq[u][t]),
                                                               acc[r][t], 0, 0, 0);
      }
      __builtin_amdgcn_sched_barrier(0);
      if (s0 + u + U < nsteps) load_step(s0 + u + U, u);
      __builtin_amdgcn_sched_barrier(0);
    }
  }
  const int N = a.N;
#pragma unroll
  for (int r = 0; r < RB; ++r) {
    if (r >= nrb) break;
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int q = 0; q < 4; ++q)
        if (wv >= QW) red[((cw * NN) + 16 * t + (lane & 15)) * 16 + 4 * (lane >> 4) + q] = acc[r][t][q];
    lds_barrier();
    // a compile-time count of slots per thread: a run-time loop here holding
    // stores would make the compiler wait for all earlier stores first
#pragma unroll
    for (int i = 0; i < (NN * 16 + NTH - 1) / NTH; ++i) {
      const int idx = tid + i * NTH;
      if (NN * 16 % NTH != 0 && idx >= NN * 16) break;
      const int row = idx & 15, node = idx >> 4;
      float sum = red[idx];
#pragma unroll
      for (int ww = 1; ww < NCW; ++ww) sum += red[ww * NN * 16 + idx];
      const int o = rbv[r] * 16 + row;
      if (node < N && o < M) {
        if constexpr (Q8) sum *= scale_r[r];
        const float y = has_bias ? sum + bf2f(bias_r[r]) : sum;
        epilogue(a, w, epi, l, node, o, y);
        if (track && (y > hb.v[i] || (y == hb.v[i] && o < hb.o[i]))) {
          hb.v[i] = y;
          hb.o[i] = o;
        }
      }
    }
    lds_barrier();
  }
  return true;
}

// one task of 1..4 row blocks, loads in flight per wave sized to the
// register budget (at four tiles one row block keeps 8 steps in flight and
// two keep 6; four row blocks keep 8 at one tile, 5 at two, 3 at four: deeper
// would spill); three code bodies serve every stage
// Runs the pre-stage (wave 0) when the workgroup has no GEMM task.
template <bool Q8, bool RE>
__device__ __forceinline__ bool pre_only(const FusedArgs& a, const Wg& w, const PreSpec& ps) {
  if (ps.kind == 0) return true;
  if (threadIdx.x < QW * 64) {
    const bool ok = do_pre<Q8, RE>(a, w, ps);
    if (threadIdx.x == 0) w.sh[0] = ok;
  }
  lds_barrier();
  const bool ok = w.sh[0] != 0;
  lds_barrier();
  return ok;
}

template <int NT, bool Q8, bool RE>
__device__ __forceinline__ bool gemm_task(const FusedArgs& a, const Wg& w, const WaitSpec& ws, int epi, int l,
                                          const int* rbs, int rb_first, int nrb, gptr<uint16_t> bias,
                                          gptr<u32x4> Wp, int KC, int M, int kc0, int kc1, const uint16_t* act,
                                          int act_kc, float* red, const PreSpec& ps, int wofs,
                                          HeadBest& hb, bool track) {
  if (nrb <= 0) return pre_only<Q8, RE>(a, w, ps);
  if (nrb == 1)
    return gemm_rb<NT, 1, NT <= 2 ? 10 : 8, Q8, RE>(a, w, ws, epi, l, rbs, rb_first, 1, bias, Wp, KC, M, kc0, kc1, act,
                                           act_kc, red, ps, wofs, hb, track);
  if (nrb == 2)
    return gemm_rb<NT, 2, NT <= 2 ? 10 : 6, Q8, RE>(a, w, ws, epi, l, rbs, rb_first, 2, bias, Wp, KC, M, kc0, kc1, act,
                                           act_kc, red, ps, wofs, hb, track);
  return gemm_rb<NT, 4, NT == 1 ? 8 : NT == 2 ? 5 : 3, Q8, RE>(a, w, ws, epi, l, rbs, rb_first, nrb, bias, Wp, KC, M, kc0,
                                                            kc1, act, act_kc, red, ps, wofs, hb, track);
}

// ------------------------------------------------------------------ tree attention
//
// Node i attends to cache rows 0..P-1 and then to its root path in the tree
// scratch (Sec. 3.1: cross-attention with the cache, self-attention in the
// batch masked by the tree).  Per (head h, 16-node tile t) the work is cut
// into units that run on different workgroups of the head's XCD:
//  * prefix unit p: cache rows 256p .. 256p + 255 (staged as K and V rows in
//    LDS).  Wave w takes rows 32w .. 32w + 31 on the matrix cores (S^T = K Q^T
//    and O^T = V^T P^T with v_mfma_f32_16x16x32_bf16; q and p as bf16 hi + lo,
//    K and V exact).  The K operand's rows are ordered so that lane l holds
//    the scores of keys 8(l/16)..+7 of node l%16, exactly its slot of the P^T
//    operand; the V^T operand is gathered from the row-major V rows.  The 8
//    waves' softmax states are merged in wave order;
//  * the root unit: each half-wave takes one node's root path on the vector
//    ALU, root first, 32 keys per batch.
// Every unit leaves a part (max, sum of exponentials, unnormalised output) per
// node; the merge stage combines a tile's parts in order (prefix parts, then
// the root path).  The cut depends on P only, so a node's result does not
// depend on the rest of the tree.

constexpr int ACH = 32 * NWV;               // prefix rows per unit: 32 per wave
static_assert(ACH == kFAttRows, "the host counts attention units of kFAttRows rows");
constexpr int AKS = DH + 8;                 // LDS row stride of K and V (elements)
constexpr int A_KV_BYTES = 2 * ACH * AKS * 2;
constexpr int A_RV_BYTES = 2 * NWV * 32 * AKS * 2;  // root-path V rows, 32 per half-wave (padded rows)
constexpr int A_REGION = A_KV_BYTES > A_RV_BYTES ? A_KV_BYTES : A_RV_BYTES;
static_assert(WST + WST_FRAGS * 1024 <= A_REGION + NWV * 16 * AREC * 4 + NWV * 2 * DH * 4,
              "staged weights must stay below the workgroup's shared words");
static_assert(WST >= (NWV - QW) * 64 * 16 * 4, "the GEMM reduction must stay below the staged weights");
constexpr int A_PART_BYTES = NWV * 16 * AREC * 4;  // the waves' states of a prefix unit
constexpr int A_Q_BYTES = NWV * 2 * DH * 4;        // root-path queries, one row per half-wave

// the part record of (head h, tile t, unit u) for tile node nl

__device__ __forceinline__ bool att_prefix_unit(const FusedArgs& a, const Wg& w, const WaitSpec& ws, int l, int h,
                                                int t, int u, unsigned char* lds) {
  uint16_t* ks = (uint16_t*)lds;
  uint16_t* vs = ks + ACH * AKS;
  float* wpart = (float*)(lds + A_REGION);  // [NWV][16][AREC]
  const int tid = opq_tid(), wv = tid >> 6, lane = tid & 63, i = lane & 15, g = lane >> 4;
  const int N = a.N, P = a.P, d = a.d;
  const float scale = a.scale;
  const size_t head_rows = ((size_t)l * a.H + h);
  const gptr<uint16_t> kc = opq(a.kc + head_rows * a.max_ctx * DH);
  const gptr<uint16_t> vc = opq(a.vc + head_rows * a.max_ctx * DH);
  const gptr<float> qbase = opq((const float*)a.q);
  const int cb = u * ACH, nk = min(ACH, P - cb);
  // The unit's cache rows do not depend on this layer's QKV outputs: waves
  // 1..7 load them before the wait (wave 0 polls, with nothing in flight).
  // Rows past the prefix re-read the last one and are zeroed below.
  constexpr int KVJ = (ACH * 8 + NTH - 64 - 1) / (NTH - 64);  // 16-byte pieces per thread
  u32x4 kr[KVJ], vr[KVJ];
  if (wv > 0) {
#pragma unroll
    for (int j = 0; j < KVJ; ++j) {
      const int e = min(tid - 64 + j * (NTH - 64), ACH * 8 - 1), r = min(e >> 3, nk - 1), c8 = e & 7;
      kr[j] = *(gptr<u32x4>)(kc + (size_t)(cb + r) * DH + 8 * c8);
      vr[j] = *(gptr<u32x4>)(vc + (size_t)(cb + r) * DH + 8 * c8);
    }
  }
  if (ws.on && !wait_flags(a, w, ws.id, ws.wx, ws.tag)) return false;
  stamp(a, w, ws.sl, ws.sfid, 1);
  // queries (B operand: node 16 t + i, dims 32 kc2 + 8 g .. +8)
  const int qn = min(16 * t + i, N - 1);
  u32x4 qh[2], ql[2];
#pragma unroll
  for (int kc2 = 0; kc2 < 2; ++kc2) {
    const gptr<float> qp = qbase + (size_t)qn * d + h * DH + 32 * kc2 + 8 * g;
    const u32x4 q0 = ld_x((gptr<u32x4>)qp), q1 = ld_x((gptr<u32x4>)(qp + 4));
    const float v[8] = {__uint_as_float(q0[0]), __uint_as_float(q0[1]), __uint_as_float(q0[2]),
                        __uint_as_float(q0[3]), __uint_as_float(q1[0]), __uint_as_float(q1[1]),
                        __uint_as_float(q1[2]), __uint_as_float(q1[3])};
    pack_hilo8(v, qh[kc2], ql[kc2]);
  }
  if (wv > 0) {
#pragma unroll
    for (int j = 0; j < KVJ; ++j) {
      const int e = tid - 64 + j * (NTH - 64), r = e >> 3, c8 = e & 7;
      if (e < ACH * 8) {
        const bool ok = r < nk;
        *(u32x4*)(ks + r * AKS + 8 * c8) = ok ? kr[j] : (u32x4){0, 0, 0, 0};
        *(u32x4*)(vs + r * AKS + 8 * c8) = ok ? vr[j] : (u32x4){0, 0, 0, 0};
      }
    }
  }
  __syncthreads();
  float m = -INFINITY, lsum = 0.f;
  f32x4 o[4];
#pragma unroll
  for (int tt = 0; tt < 4; ++tt) o[tt] = (f32x4){0.f, 0.f, 0.f, 0.f};
  if (32 * wv < nk) {
    const uint16_t* kb = ks + (32 * wv + 8 * (i >> 2) + (i & 3)) * AKS + 8 * g;
    f32x4 s0 = (f32x4){0, 0, 0, 0}, s1 = (f32x4){0, 0, 0, 0};
#pragma unroll
    for (int kc2 = 0; kc2 < 2; ++kc2) {
      const u32x4 k0 = *(const u32x4*)(kb + 32 * kc2);
      const u32x4 k1 = *(const u32x4*)(kb + 4 * AKS + 32 * kc2);
      s0 = mfma_bf16(k0, qh[kc2], s0);
      s0 = mfma_bf16(k0, ql[kc2], s0);
      s1 = mfma_bf16(k1, qh[kc2], s1);
      s1 = mfma_bf16(k1, ql[kc2], s1);
    }
    float sv[8];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int key = 32 * wv + 8 * g + r;
      sv[r] = key < nk ? s0[r] * scale : -INFINITY;
      sv[4 + r] = key + 4 < nk ? s1[r] * scale : -INFINITY;
    }
    float mb = sv[0];
#pragma unroll
    for (int e = 1; e < 8; ++e) mb = fmaxf(mb, sv[e]);
    mb = fmaxf(mb, __shfl_xor(mb, 16));
    mb = fmaxf(mb, __shfl_xor(mb, 32));
    m = mb;
    float pv[8], ps = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      pv[e] = __expf(sv[e] - m);
      ps += pv[e];
    }
    ps += __shfl_xor(ps, 16);
    ps += __shfl_xor(ps, 32);
    lsum = ps;
    u32x4 ph, pl;
    pack_hilo8(pv, ph, pl);
#pragma unroll
    for (int tt = 0; tt < 4; ++tt) {
      // A operand V^T (16 dims x 32 keys): lane (i, g) gathers dim 16 tt + i
      // of keys 8 g .. 8 g + 7 of this wave's 32 from the row-major rows
      const uint16_t* vcol = vs + (32 * wv + 8 * g) * AKS + 16 * tt + i;
      uint32_t hh[8];
#pragma unroll
      for (int jj = 0; jj < 8; ++jj) hh[jj] = vcol[jj * AKS];
      const u32x4 va = (u32x4){hh[0] | (hh[1] << 16), hh[2] | (hh[3] << 16), hh[4] | (hh[5] << 16),
                               hh[6] | (hh[7] << 16)};
      o[tt] = mfma_bf16(va, ph, o[tt]);
      o[tt] = mfma_bf16(va, pl, o[tt]);
    }
  }
  // this wave's state of node 16 t + i: lane (i, g) holds dims 16 tt + 4 g + r
  {
    float* rec = wpart + (wv * 16 + i) * AREC;
    if (g == 0) {
      rec[0] = m;
      rec[1] = lsum;
    }
#pragma unroll
    for (int tt = 0; tt < 4; ++tt) *(f32x4*)(rec + 4 + 16 * tt + 4 * g) = o[tt];
  }
  lds_barrier();
  // the waves merged in wave order into the unit's part: thread -> node,
  // DPT consecutive dims
  {
    constexpr int DPT = 16 * DH / NTH;
    const int nl = tid / (DH / DPT), d0 = DPT * (tid % (DH / DPT));
    float M = -INFINITY, L = 0.f, O[DPT];
#pragma unroll
    for (int e = 0; e < DPT; ++e) O[e] = 0.f;
    // every wave's state read at once (one LDS round trip), then merged in
    // wave order; a wave with no keys (max -inf) is skipped
    float mv[NWV], lv[NWV], ovv[NWV][DPT];
#pragma unroll
    for (int j = 0; j < NWV; ++j) {
      const float* rec = wpart + (j * 16 + nl) * AREC;
      mv[j] = rec[0];
      lv[j] = rec[1];
#pragma unroll
      for (int e = 0; e < DPT; ++e) ovv[j][e] = rec[4 + d0 + e];
    }
#pragma unroll
    for (int j = 0; j < NWV; ++j) {
      if (mv[j] == -INFINITY) continue;
      const float mn = fmaxf(M, mv[j]);
      const float al = __expf(M - mn), wj = __expf(mv[j] - mn);
      L = fmaf(L, al, lv[j] * wj);
#pragma unroll
      for (int e = 0; e < DPT; ++e) O[e] = fmaf(O[e], al, ovv[j][e] * wj);
      M = mn;
    }
    const gw<float> out = part_rec(a, h, t, u, nl);
    if (d0 == 0) {
      out[0] = M;
      out[1] = L;
    }
#pragma unroll
    for (int e = 0; e < DPT; ++e) out[4 + d0 + e] = O[e];
  }
  lds_barrier();  // LDS is reused by the next unit; the stores are waited for by unit_done
  return true;
}

__device__ __forceinline__ bool att_root_unit(const FusedArgs& a, const Wg& w, const WaitSpec& ws, int l, int h,
                                              int t, unsigned char* lds) {
  float* qrow = (float*)(lds + A_REGION + A_PART_BYTES);  // [NWV][2][DH]
  const int tid = opq_tid(), wv = tid >> 6, lane = tid & 63;
  const int N = a.N, d = a.d;
  const float scale = a.scale;
  const size_t head_rows = ((size_t)l * a.H + h);
  const gptr<float> qbase = opq((const float*)a.q);
  const gptr<int> tree = opq(a.tree);
  constexpr int DPL = DH / 32;  // dims per lane of a half-wave
  const int hw = lane >> 5, hl = lane & 31;
  const gptr<int> depth = tree + 2 * a.max_nodes;
  const gptr<int> anc_off = tree + 4 * a.max_nodes;
  const gptr<int> path32 = tree + 5 * a.max_nodes;
  const gptr<int> ancl = path32 + (size_t)N * kPath32;
  const int nl = 2 * wv + hw;  // this half-wave's node within the tile
  const int rnc = min(16 * t + nl, N - 1);
  // the tree's indices are known before this layer's QKV outputs are
  int rkey = ld_x(path32 + (size_t)rnc * kPath32 + hl);
  const int rdep = ld_x(depth + rnc);
  if (ws.on && !wait_flags(a, w, ws.id, ws.wx, ws.tag)) return false;
  stamp(a, w, ws.sl, ws.sfid, 1);
  const gptr<uint16_t> ktb = opq((const uint16_t*)a.kt + head_rows * a.max_nodes * DH);
  const gptr<uint16_t> vtb = opq((const uint16_t*)a.vt + head_rows * a.max_nodes * DH);
  u32x4 rk[DH / 8], rv[DH / 8];
#pragma unroll
  for (int j = 0; j < DH / 8; ++j) {
    rk[j] = ld_x((gptr<u32x4>)(ktb + (size_t)rkey * DH + 8 * j));
    rv[j] = ld_x((gptr<u32x4>)(vtb + (size_t)rkey * DH + 8 * j));
  }
  uint16_t* rvl = (uint16_t*)lds + (2 * wv + hw) * 32 * AKS;  // [32 keys][AKS]: padded, conflict-free
  float* qr = qrow + (wv * 2 + hw) * DH;
  {
    const gptr<float> qp = qbase + (size_t)rnc * d + h * DH + hl * DPL;
#pragma unroll
    for (int e = 0; e < DPL; ++e) qr[hl * DPL + e] = ld_x(qp + e);
  }
  float rm = -INFINITY, rl = 0.f, ro[DPL];
#pragma unroll
  for (int e = 0; e < DPL; ++e) ro[e] = 0.f;
  const int rbatches = (max(rdep, __shfl_xor(rdep, 32)) + 32) / 32;  // wave-uniform
  for (int bt = 0; bt < rbatches; ++bt) {
    const int j = 32 * bt + hl;
    if (bt > 0) {
      rkey = ld_x(ancl + ld_x(anc_off + rnc) + min(j, rdep));
#pragma unroll
      for (int jj = 0; jj < DH / 8; ++jj) {
        rk[jj] = ld_x((gptr<u32x4>)(ktb + (size_t)rkey * DH + 8 * jj));
        rv[jj] = ld_x((gptr<u32x4>)(vtb + (size_t)rkey * DH + 8 * jj));
      }
    }
#pragma unroll
    for (int jj = 0; jj < DH / 8; ++jj) *(u32x4*)(rvl + hl * AKS + 8 * jj) = rv[jj];
    wave_sync_lds();
    // four independent chains over the dims, combined in a fixed order
    float dq[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int c8 = 0; c8 < DH / 8; ++c8) {
      const f32x4 qa = *(const f32x4*)&qr[8 * c8];
      const f32x4 qb = *(const f32x4*)&qr[8 * c8 + 4];
      const u32x4 ku = rk[c8];
      float& d0 = dq[(2 * c8) & 3];
      float& d1 = dq[(2 * c8 + 1) & 3];
      d0 = fmaf(qa[0], __uint_as_float(ku[0] << 16), d0);
      d0 = fmaf(qa[1], __uint_as_float(ku[0] & 0xffff0000u), d0);
      d0 = fmaf(qa[2], __uint_as_float(ku[1] << 16), d0);
      d0 = fmaf(qa[3], __uint_as_float(ku[1] & 0xffff0000u), d0);
      d1 = fmaf(qb[0], __uint_as_float(ku[2] << 16), d1);
      d1 = fmaf(qb[1], __uint_as_float(ku[2] & 0xffff0000u), d1);
      d1 = fmaf(qb[2], __uint_as_float(ku[3] << 16), d1);
      d1 = fmaf(qb[3], __uint_as_float(ku[3] & 0xffff0000u), d1);
    }
    const float dot = (dq[0] + dq[1]) + (dq[2] + dq[3]);
    const bool kvalid = j <= rdep;
    const float sc = kvalid ? dot * scale : -INFINITY;
    const float mb = half_max(sc);
    const float mn = fmaxf(rm, mb);
    const float alpha = __expf(rm - mn);
    const float p = kvalid ? __expf(sc - mn) : 0.f;
    const float ps = half_sum(p);
    rl = fmaf(rl, alpha, ps);
    rm = mn;
    const int cnt = min(32, rdep + 1 - 32 * bt);
    const int cmax = max(cnt, __shfl_xor(cnt, 32));  // wave-uniform
    float acc[DPL];
#pragma unroll
    for (int e = 0; e < DPL; ++e) acc[e] = 0.f;
    for (int jj = 0; jj < cmax; ++jj) {
      const float pj = jj < cnt ? __shfl(p, (hw << 5) + jj) : 0.f;
      const uint16_t* vr2 = rvl + jj * AKS + DPL * hl;
#pragma unroll
      for (int e = 0; e < DPL; ++e) acc[e] = fmaf(pj, bf2f(vr2[e]), acc[e]);
    }
#pragma unroll
    for (int e = 0; e < DPL; ++e) ro[e] = fmaf(ro[e], alpha, acc[e]);
    wave_sync_lds();
  }
  const gw<float> out = part_rec(a, h, t, a.att_units, nl);
  if (hl == 0) {
    out[0] = rm;
    out[1] = rl;
  }
#pragma unroll
  for (int e = 0; e < DPL; ++e) out[4 + DPL * hl + e] = ro[e];
  lds_barrier();  // LDS is reused by the next unit; the stores are waited for by unit_done
  return true;
}

// the merge of (head h, tile t): prefix parts in order, then the root path,
// written as the out-projection's float16 input
// ------------------------------------------------------------------ the plan of one workgroup
//
// int32 [kPlanStride] per workgroup (see FusedPlan in ssd_internal.h):
//   ATT: count, then head | tile << 16
//   QKV, WO, FC, WPR: count, then row blocks
//   HEAD: first row block, end row block of the LM head

// ------------------------------------------------------------------ compute workgroups

template <int NT, bool Q8, bool RE>
__device__ __forceinline__ void compute_wg(const FusedArgs& a, unsigned char* lds) {
  int* sh = (int*)(lds + A_REGION + A_PART_BYTES + A_Q_BYTES);  // 32 words
  int* lplan = sh + 32;                                            // [kPlanStride]
  unsigned long long* llw = (unsigned long long*)(lplan + kPlanStride);  // [L][kLwSlots]
  float* red = (float*)lds;                                        // GEMM / LN reductions
  Wg w;
  w.x = (int)xcc_id();
  w.r = blockIdx.x >> 3;
  w.g = w.x * kFRanks + w.r;
  w.sh = sh;
  w.lds = lds;
  w.plan = lplan;
  w.lwt = llw;
  {
    const int g = w.x * kFRanks + w.r;
    if (threadIdx.x < kPlanStride && w.x < kFXcd) lplan[threadIdx.x] = a.plan[(size_t)g * kPlanStride + threadIdx.x];
    for (int i = threadIdx.x; i < a.L * kLwSlots; i += NTH) llw[i] = (unsigned long long)a.lw[i];
  }
  if (threadIdx.x == 0) {
    const unsigned E = __hip_atomic_load(&a.ctl[FZ_PASS], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) + 1u;
    sh[1] = (int)E;
    // (x, r) must name one workgroup of 8 XCDs: a second claim in the same pass aborts
    int ok = w.x < kFXcd;
    if (ok) ok = __hip_atomic_exchange(&a.ctl[FZ_CLAIM + w.g], E, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != E;
    if (!ok) raise_abort(a, 1u);
    sh[3] = ok;
    sh[4] = 0;  // the counter of q_barrier
  }
  __syncthreads();
  w.E = (unsigned)sh[1];
  w.tagbase = w.E * kFTagsPerPass;
  const bool placed = sh[3] != 0;
  __syncthreads();
  if (!placed) {
    // not a valid (XCD, rank): count as finished, touch nothing else
    if (threadIdx.x == 0) {
      const unsigned prev = __hip_atomic_fetch_add(&a.ctl[FZ_DONE], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      if (prev == kFGroups - 1) {
        __hip_atomic_store(&a.ctl[FZ_DONE], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_store(&a.ctl[FZ_ABORT], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_store(&a.ctl[FZ_PASS], w.E, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
    }
    return;
  }

  // Rank 0 of each XCD clears the tile counters of the XCD's heads (a pass
  // that ended early may have left counts behind).  Its stores complete
  // before its first stage flag, and every attention unit of the XCD waits
  // for that rank's QKV flag, so the counters are 0 before any unit counts.
  if (w.r == 0 && (int)threadIdx.x < 4 * (a.xh[2 * w.x + 1] - a.xh[2 * w.x]))
    __hip_atomic_store(a.tile_ctr + (size_t)a.xh[2 * w.x] * 4 + threadIdx.x, 0u, __ATOMIC_RELAXED,
                       __HIP_MEMORY_SCOPE_AGENT);
  const int* p = w.plan;
  const int n_qkv = p[PL_QKV], n_wo = p[PL_WO], n_fc = p[PL_FC], n_wpr = p[PL_WPR];
  const int hb0 = p[PL_HEAD], hb1 = p[PL_HEAD + 1];
  const int d = a.d, M = a.M, KCd = d / 32, KCm = M / 32;
  const int kh0 = 2 * a.xh[2 * w.x], kh1 = 2 * a.xh[2 * w.x + 1];  // the XCD's heads, in k-steps of W_o
  const int kf0 = a.xf[2 * w.x], kf1 = a.xf[2 * w.x + 1];           // hidden slice, in k-steps of W_pr
  uint16_t* act1 = a.act1 + (size_t)w.x * a.act_stride;
  uint16_t* act2 = a.act2 + (size_t)w.x * a.act_stride;
  const int N = a.N, L = a.L;

  // One runtime loop over the pass's stages, so that each stage body (the
  // LayerNorm, the GEMM at 1, 2 and 4 row blocks, the attention units)
  // exists once in the code.
  //   kind 0..7: LN1, QKV, ATT, (3: none; the last attention unit of a
  //   tile merges it), WO, LN2, FC, WPR of layer l; 8: final LayerNorm; 9:
  //   LM head.  Kinds 1, 6 and 9 run in the same iteration as the
  //   LayerNorm before them.
  const int NTl = (N + 15) / 16;             // 16-node tiles
  const int S = a.att_units;                 // prefix units of 256 cache rows
  const int nhx = a.xh[2 * w.x + 1] - a.xh[2 * w.x];
  const int n_attu = nhx * NTl * (S + 1);    // attention units of this XCD (prefix units + root unit per tile)
  // With two or more node tiles, the MLP down-projection's weights are
  // copied into LDS during the up-projection (by waves 1..3, which ran the
  // LayerNorm) when they fit.  The up-projection's closing wait covers the
  // copy; with one tile that stage is too short to hide it.
  const bool wpr_staged = NT >= 2 && n_wpr > 0 && n_wpr * (kf1 - kf0) <= WST_FRAGS;
  const bool wpr_early = wpr_staged && NT == 4;  // (see the out-projection stage)
  // likewise the out-projection's weights during LN1 + QKV, above the
  // parameter table (the attention stage between uses the LDS below it)
  const int wo_ofs = A_REGION + A_PART_BYTES + A_Q_BYTES + 256 + L * kLwSlots * 8;
  const bool wo_staged = NT >= 2 && n_wo > 0 && n_wo * (kh1 - kh0) <= WO_FRAGS;
  HeadBest hbest{{-INFINITY, -INFINITY}, {0x7fffffff, 0x7fffffff}};
  const int nst = L * 8 + 2, L0 = RE ? a.l0 : 0;  // (L0: the first layer this pass runs)
  for (int st = L0 * 8; st < nst; ++st) {
    const int l = st < L * 8 ? st / 8 : L;
    const int kind = st < L * 8 ? st % 8 : 8 + (st - L * 8);
    if (kind == 1 || kind == 3 || kind == 6 || kind == 9) continue;  // run with the stage before them, or none
    if (kind == 2) {
      // attention units of this XCD's heads, dealt to its ranks in turn
      stamp(a, w, l, FS_ATT, 0);
      const WaitSpec ws{FS_QKV, w.x, tag_of(w, l, FS_QKV), true, l, FS_ATT};
      const WaitSpec none{0, 0, 0u, false, l, FS_ATT};
      // units go to the ranks in the plan's order (fewest QKV row blocks
      // first: they are the first to be free)
      const int apos = p[PL_ATT];
      for (int u = apos; u < n_attu; u += kFRanks) {
        // units in (head, tile, part) order; when they outnumber the ranks,
        // the root units of every (head, tile) first, so that the ranks that
        // take a second unit took a (shorter) root unit first (measured: 1.5 %
        // faster at 64 nodes; at 16 and 32 nodes the plain order is faster)
        int hloc, t, part;
        if (n_attu <= kFRanks) {
          hloc = u / (NTl * (S + 1));
          const int rem = u - hloc * (NTl * (S + 1));
          t = rem / (S + 1);
          part = rem - t * (S + 1);
        } else if (u < nhx * NTl) {
          hloc = u / NTl;
          t = u - hloc * NTl;
          part = S;
        } else {
          const int v = u - nhx * NTl;
          hloc = v / (NTl * S);
          const int rem = v - hloc * (NTl * S);
          t = rem / S;
          part = rem - t * S;
        }
        const int h = a.xh[2 * w.x] + hloc;
        const WaitSpec& wsu = u == apos ? ws : none;
        const bool ok = part < S ? att_prefix_unit(a, w, wsu, l, h, t, part, lds)
                                 : att_root_unit(a, w, wsu, l, h, t, lds);
        if (!ok) goto out;
        unit_done(a, w, l, h, t, part);
      }
      signal(a, w, l, FS_ATT, false);
      stamp(a, w, l, FS_ATT, 2);
      continue;
    }
    if (kind == 4 || kind == 7) {
      // the residual GEMMs: out-projection over this XCD's heads (the merged
      // attention output), MLP down-projection over its hidden slice; both
      // leave partial residuals for every XCD's next LayerNorm
      const bool wo = kind == 4;
      const int fid = wo ? FS_WO : FS_WPR;
      stamp(a, w, l, fid, 0);
      const WaitSpec ws{wo ? FS_ATT : FS_FC, w.x, tag_of(w, l, wo ? FS_ATT : FS_FC), true, l, fid};
      PreSpec nopre{};
      const bool ok = wo ? gemm_task<NT, Q8, RE>(a, w, ws, FE_WO, l, p + PL_WO + 1, 0, n_wo, G<uint16_t>(nullptr),
                                         G<u32x4>(lw(w, l, LW_O)), KCd, d, kh0, kh1, a.fo, KCd, red, nopre,
                                         wo_staged ? wo_ofs : 0, hbest, false)
                         : gemm_task<NT, Q8, RE>(a, w, ws, FE_WPR, l, p + PL_WPR + 1, 0, n_wpr, G<uint16_t>(nullptr),
                                         G<u32x4>(lw(w, l, LW_PR)), KCm, d, kf0, kf1, a.ff, KCm, red, nopre,
                                         wpr_staged ? WST : 0, hbest, false);
      if (!ok) goto out;
      signal(a, w, l, fid, true);
      stamp(a, w, l, fid, 2);
      if (wo && wpr_early && threadIdx.x >= 64) {
        // at four node tiles the down-projection's weights are copied into
        // LDS from here (waves 1..7), inside the LayerNorm's cross-XCD wait,
        // rather than after the LayerNorm's rows (measured: 3 % faster at
        // 64 nodes, neutral or slower at 32)
        stage_frags<Q8>(G<u32x4>(lw(w, l, LW_PR)), p + PL_WPR + 1, n_wpr, kf0, kf1 - kf0, KCm, lds + WST,
                        threadIdx.x >> 6, NWV - 1);
      }
      continue;
    }
    // kind 0, 5, 8: waves 0..3 run this LayerNorm stage while waves 4..7
    // already load the weights of the GEMM stage that follows it (QKV, MLP
    // up-projection, LM head), which the workgroup then runs.
    PreSpec ps{};
    ps.l = l;
    ps.kind = 1;
    ps.fid = kind == 5 ? FS_LN2 : FS_LN1;
    ps.mode = (kind == 0 && l == L0) ? 0 : 1;
    if (kind == 5) {
      if (wpr_staged && !wpr_early) {
        ps.wn = n_wpr;
        ps.wk0 = kf0;
        ps.wk1 = kf1;
        ps.wKC = KCm;
        ps.wdst = WST;
        ps.wrbs = p + PL_WPR + 1;
        ps.wW = G<u32x4>(lw(w, l, LW_PR));
      }
      ps.ws = WaitSpec{FS_WO, -1, tag_of(w, l, FS_WO), true, l, FS_LN2};
      ps.bias = G<uint16_t>(lw(w, l, LB_O));
      ps.kin = 2 * l;
      ps.zmask = 1u << ((2 * l + 2) % 3);  // sub-layer 2l - 1's buffer
      ps.g = G<uint16_t>(lw(w, l, LN2G));
      ps.b = G<uint16_t>(lw(w, l, LN2B));
      ps.act = act2;
    } else {
      if (kind == 0 && wo_staged) {
        ps.wn = n_wo;
        ps.wk0 = kh0;
        ps.wk1 = kh1;
        ps.wKC = KCd;
        ps.wdst = wo_ofs;
        ps.wrbs = p + PL_WO + 1;
        ps.wW = G<u32x4>(lw(w, l, LW_O));
      }
      const int lp = kind == 8 ? L - 1 : max(l - 1, 0);
      ps.ws = WaitSpec{FS_WPR, -1, tag_of(w, lp, FS_WPR), kind == 8 || l > L0, l, FS_LN1};
      ps.bias = G<uint16_t>(lw(w, lp, LB_PR));
      ps.kin = 2 * lp + 1;
      // sub-layer 2lp's buffer; the pass's first layer clears the two its
      // own sub-layers add into
      ps.zmask = ps.mode == 0 ? (1u << ((2 * l) % 3)) | (1u << ((2 * l + 1) % 3)) : 1u << ((2 * lp) % 3);
      ps.g = kind == 8 ? G<uint16_t>(a.lnf_g) : G<uint16_t>(lw(w, l, LN1G));
      ps.b = kind == 8 ? G<uint16_t>(a.lnf_b) : G<uint16_t>(lw(w, l, LN1B));
      ps.act = act1;
    }
    stamp(a, w, l, ps.fid, 0);
    int gfid, epi, nrb, Mo, k0 = 0, k1 = KCd, rb_first = 0;
    const int* rbs = nullptr;
    gptr<uint16_t> bias = G<uint16_t>(nullptr);
    gptr<u32x4> Wm;
    const uint16_t* act = act1;
    switch (kind) {
      case 0: gfid = FS_QKV; epi = FE_QKV; nrb = n_qkv; rbs = p + PL_QKV + 1; Wm = G<u32x4>(lw(w, l, LW_QKV));
              Mo = 3 * d; bias = G<uint16_t>(lw(w, l, LB_QKV)); break;
      case 5: gfid = FS_FC; epi = FE_FC; nrb = n_fc; rbs = p + PL_FC + 1; Wm = G<u32x4>(lw(w, l, LW_FC)); Mo = M;
              bias = G<uint16_t>(lw(w, l, LB_FC)); act = act2; break;
      default: gfid = FS_QKV; epi = FE_HEAD; nrb = min(4, hb1 - hb0); rb_first = hb0; Wm = G<u32x4>(a.p_head);
               Mo = a.V; break;
    }
    {
      // (the first QKV stage waits for every XCD's first LayerNorm, which
      // clears the first two sum buffers: see xs_zero)
      const WaitSpec gws{ps.fid, (kind == 0 && l == L0) ? -1 : w.x, tag_of(w, l, ps.fid), true, l, gfid};
      if (!gemm_task<NT, Q8, RE>(a, w, gws, epi, l, rbs, rb_first, nrb, bias, Wm, KCd, Mo, k0, k1, act, KCd, red, ps, 0,
                         hbest, kind == 8))
        goto out;
    }
    if (kind == 8) {
      // the rest of this workgroup's LM-head row blocks, 4 at a time
      const WaitSpec none{0, 0, 0u, false, l, gfid};
      PreSpec nopre{};
      for (int b0 = hb0 + 4, j = 1; b0 < hb1; b0 += 4, ++j) {
        if (!gemm_task<NT, Q8, RE>(a, w, none, FE_HEAD, L, nullptr, b0, min(4, hb1 - b0), G<uint16_t>(nullptr),
                           G<u32x4>(a.p_head), KCd, a.V, 0, KCd, act1, KCd, red, nopre, 0, hbest, true))
          goto out;
      }
      // this workgroup's maximum per node: the 16 slots of a node sit in 16
      // consecutive lanes; (logit, token) pairs, ties to the lower token
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        float v = hbest.v[i];
        int o = hbest.o[i];
#pragma unroll
        for (int m = 1; m < 16; m <<= 1) {
          const float v2 = __shfl_xor(v, m);
          const int o2 = __shfl_xor(o, m);
          if (v2 > v || (v2 == v && o2 < o)) {
            v = v2;
            o = o2;
          }
        }
        const int idx = threadIdx.x + i * NTH, node = idx >> 4;
        if ((idx & 15) == 0 && idx < 16 * 16 * NT && node < N)
          *(gw<u32x2>)(a.head_part + ((size_t)node * kFGroups + w.g) * 2) = (u32x2){__float_as_uint(v), (unsigned)o};
      }
    }
    signal(a, w, l, gfid, false);
    stamp(a, w, l, gfid, 2);
  }
out:
  __syncthreads();
  if (threadIdx.x == 0) {
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    const unsigned prev = __hip_atomic_fetch_add(&a.ctl[FZ_DONE], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (prev == kFGroups - 1) {
      __hip_atomic_store(&a.ctl[FZ_DONE], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(&a.ctl[FZ_ABORT], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(&a.ctl[FZ_PASS], w.E, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
}


// RE: the pass starts at layer a.l0 from the residual stream a.x_in
template <int NT, bool Q8, bool RE>
__global__ __launch_bounds__(NTH) __attribute__((amdgpu_waves_per_eu(2))) void pass_kernel(FusedArgs a) {
  extern __shared__ __attribute__((aligned(16))) unsigned char lds[];
  compute_wg<NT, Q8, RE>(a, lds);
}

}  // namespace fz

// ------------------------------------------------------------------ host planner
//
// Splits one layer over the 8 XCDs and their 32 ranks.
//  * Heads: the first H % 8 XCDs take one more.  A head costs 4 x 64 rows of
//    d weights (Q, K, V rows and the W_o columns); a hidden feature costs 2 d.
//    Each XCD's hidden slice (whole k-steps of 32 features) is chosen so that
//    every XCD streams about the same bytes per layer.
//  * Inside an XCD each stage's units (attention head x tile; row blocks of
//    the GEMMs) are dealt so that every rank gets floor or ceil of its share
//    of that stage, the extra units going to the ranks with the least bytes
//    so far; a rank's units of a stage are consecutive.
//  * The LM head's row blocks are cut into 256 consecutive ranges.
bool fused_plan(int H, int d, int M, int V, int ntiles, int* tab, int* xh, int* xf, std::string* why) {
  const int DHh = 64;
  if (H * DHh != d || d % 32 || M % 32 || ntiles < 1 || ntiles > 4) {
    *why = "fused pass: needs head dimension 64, d and d_mlp multiples of 32, 1-4 node tiles";
    return false;
  }
  const int KM = M / 32;
  int hx[kFXcd], fx[kFXcd];
  for (int x = 0; x < kFXcd; ++x) hx[x] = H / kFXcd + (x < H % kFXcd ? 1 : 0);
  // bytes per layer in units of 4 d bytes: 128 per head, 1 per hidden feature
  const double target = (128.0 * H + M) / kFXcd;
  int fsum = 0;
  for (int x = 0; x < kFXcd; ++x) {
    const double want = (target - 128.0 * hx[x]) / 32.0;
    fx[x] = want > 0 ? (int)want : 0;
    fsum += fx[x];
  }
  auto load = [&](int x) { return 128.0 * hx[x] + 32.0 * fx[x]; };
  while (fsum < KM) {
    int b = 0;
    for (int x = 1; x < kFXcd; ++x)
      if (load(x) < load(b)) b = x;
    ++fx[b];
    ++fsum;
  }
  while (fsum > KM) {
    int b = -1;
    for (int x = 0; x < kFXcd; ++x)
      if (fx[x] > 0 && (b < 0 || load(x) > load(b))) b = x;
    --fx[b];
    --fsum;
  }
  int h0 = 0, f0 = 0;
  for (int x = 0; x < kFXcd; ++x) {
    xh[2 * x] = h0;
    xh[2 * x + 1] = h0 + hx[x];
    h0 += hx[x];
    xf[2 * x] = f0;
    xf[2 * x + 1] = f0 + fx[x];
    f0 += fx[x];
  }
  std::fill(tab, tab + (size_t)kFGroups * kPlanStride, 0);
  const int RBd = d / 16;
  for (int x = 0; x < kFXcd; ++x) {
    std::vector<int> unitsQ, unitsO, unitsF, unitsP;
    for (int part = 0; part < 3; ++part)
      for (int h = xh[2 * x]; h < xh[2 * x + 1]; ++h)
        for (int j = 0; j < DHh / 16; ++j) unitsQ.push_back(part * RBd + h * (DHh / 16) + j);
    if (hx[x] > 0)
      for (int rb = 0; rb < RBd; ++rb) unitsO.push_back(rb);
    for (int rb = 2 * xf[2 * x]; rb < 2 * xf[2 * x + 1]; ++rb) unitsF.push_back(rb);
    if (fx[x] > 0)
      for (int rb = 0; rb < RBd; ++rb) unitsP.push_back(rb);
    // Ranks finishing a stage early start the next one early, so each
    // stage's extra units go to the ranks with the least work in the stage
    // before it (stable: lower ranks first among equals).
    std::vector<double> prev(kFRanks, 0.0);
    auto order_by_prev = [&]() {
      std::vector<int> order(kFRanks);
      for (int r = 0; r < kFRanks; ++r) order[r] = r;
      std::stable_sort(order.begin(), order.end(), [&](int p, int q) { return prev[p] < prev[q]; });
      return order;
    };
    auto deal = [&](const std::vector<int>& u, int slot, double cost) {
      const int U = (int)u.size(), base = U / kFRanks, extra = U % kFRanks;
      const std::vector<int> order = order_by_prev();
      std::vector<int> cnt(kFRanks, base);
      for (int k = 0; k < extra; ++k) cnt[order[k]]++;
      int next = 0;
      for (int r = 0; r < kFRanks; ++r) {
        if (cnt[r] > kPlanMaxRb) return false;
        int* row = tab + (size_t)(x * kFRanks + r) * kPlanStride;
        row[slot] = cnt[r];
        for (int k = 0; k < cnt[r]; ++k) row[slot + 1 + k] = u[next++];
        prev[r] = cnt[r] * cost;
      }
      return true;
    };
    bool ok = deal(unitsQ, PL_QKV, 32.0 * d);
    // attention: units u = pos, pos + 32, ... go to the rank at position pos
    // of this order (its cost taken at a nominal 512-row prefix: 3 units per
    // head and tile)
    const std::vector<int> aorder = order_by_prev();
    const int n_att = 3 * hx[x] * ntiles;
    for (int pos = 0; pos < kFRanks; ++pos) {
      const int r = aorder[pos];
      tab[(size_t)(x * kFRanks + r) * kPlanStride + PL_ATT] = pos;
      prev[r] = (double)((n_att - pos + kFRanks - 1) / kFRanks) * 256.0 * 256.0;
    }
    ok = ok && deal(unitsO, PL_WO, 16.0 * 64 * hx[x] * 2);
    std::fill(prev.begin(), prev.end(), 0.0);  // LN2: one node row per rank, evenly
    ok = ok && deal(unitsF, PL_FC, 32.0 * d);
    ok = ok && deal(unitsP, PL_WPR, 16.0 * 32 * fx[x] * 2);
    if (!ok) {
      *why = "fused pass: a rank would get more than the plan's units per stage";
      return false;
    }
  }
  const int RBV = (V + 15) / 16;
  for (int g = 0; g < kFGroups; ++g) {
    int* row = tab + (size_t)g * kPlanStride;
    row[PL_HEAD] = (int)((long long)g * RBV / kFGroups);
    row[PL_HEAD + 1] = (int)((long long)(g + 1) * RBV / kFGroups);
  }
  return true;
}

hipError_t fused_prepare() {
  const int lds = (int)fused_lds_bytes(kFMaxL);
  const void* fns[] = {
      (const void*)fz::pass_kernel<1, false, false>, (const void*)fz::pass_kernel<2, false, false>,
      (const void*)fz::pass_kernel<4, false, false>, (const void*)fz::pass_kernel<1, true, false>,
      (const void*)fz::pass_kernel<2, true, false>,  (const void*)fz::pass_kernel<4, true, false>,
      (const void*)fz::pass_kernel<1, false, true>,  (const void*)fz::pass_kernel<2, false, true>,
      (const void*)fz::pass_kernel<4, false, true>,  (const void*)fz::pass_kernel<1, true, true>,
      (const void*)fz::pass_kernel<2, true, true>,   (const void*)fz::pass_kernel<4, true, true>};
  hipError_t e = hipSuccess;
  for (size_t i = 0; i < sizeof(fns) / sizeof(fns[0]) && e == hipSuccess; ++i)
    e = hipFuncSetAttribute(fns[i], hipFuncAttributeMaxDynamicSharedMemorySize, lds);
  return e;
}

// attention / GEMM regions, shared words, plan row, the layers' parameter
// pointers, the out-projection's staged weights
size_t fused_lds_bytes(int L) {
  return fz::A_REGION + fz::A_PART_BYTES + fz::A_Q_BYTES + 128 + kPlanStride * 4 + (size_t)L * kLwSlots * 8 +
         fz::WO_FRAGS * 1024;
}
static_assert(fz::A_REGION + fz::A_PART_BYTES + fz::A_Q_BYTES + 128 + kPlanStride * 4 + kFMaxL * kLwSlots * 8 +
                      fz::WO_FRAGS * 1024 <= 160 * 1024,
              "the persistent pass's LDS must fit a gfx950 workgroup (160 KB)");

template <bool Q8, bool RE>
static void launch_tiles(const FusedArgs& a, int nt, dim3 grid, size_t lds, hipStream_t s) {
  switch (nt) {
    case 1: fz::pass_kernel<1, Q8, RE><<<grid, fz::NTH, lds, s>>>(a); break;
    case 2: fz::pass_kernel<2, Q8, RE><<<grid, fz::NTH, lds, s>>>(a); break;
    default: fz::pass_kernel<4, Q8, RE><<<grid, fz::NTH, lds, s>>>(a); break;
  }
}

hipError_t launch_fused(const FusedArgs& a, hipStream_t s) {
  if (a.N <= 0 || a.N > kFMaxN || a.d % 32 || a.M % 32 || a.d > 2048 || a.H * fz::DH != a.d) return hipErrorInvalidValue;
  if (a.l0 < 0 || a.l0 >= a.L || (a.l0 > 0 && !a.x_in)) return hipErrorInvalidValue;
  const int nt = (a.N + 15) / 16;
  const size_t lds = fused_lds_bytes(a.L);
  const dim3 grid(kFGroups);
  // (the variants: 16- or 8-bit weights, a pass from the embedding or from
  // a later layer's residual stream)
  if (a.q8) {
    if (a.l0 > 0) launch_tiles<true, true>(a, nt, grid, lds, s);
    else launch_tiles<true, false>(a, nt, grid, lds, s);
  } else {
    if (a.l0 > 0) launch_tiles<false, true>(a, nt, grid, lds, s);
    else launch_tiles<false, false>(a, nt, grid, lds, s);
  }
  return hipGetLastError();
}

}  // namespace ssd
