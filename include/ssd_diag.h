/*
 * ssd_diag.h — measurement and diagnostic entry points of libssd.
 *
 * Not part of the method's interface (ssd.h): these expose internals of the
 * verification pass so that benchmarks and tests can time one kernel alone,
 * check the persistent launch's work split on the host, or record its stage
 * timestamps.  Same conventions as ssd.h.
 */
#ifndef SSD_DIAG_H
#define SSD_DIAG_H

#include "ssd.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Launches one weight GEMM of the verification pass on its own, exactly as
 * the pass launches it, for measurement: which = 0 QKV, 1 attention output,
 * 2 MLP up (FC + GELU), 3 MLP down; layer in [0, n_layer).  Reads and writes
 * only the session's workspaces and tree scratch (never the cache or caller
 * buffers), so results are meaningless outside a pass. */
ssd_status ssd_launch_gemm(const ssd_model *m, ssd_kv *kv, int32_t which, int32_t layer, int32_t n_nodes,
                           void *stream);

/* Host-only: which way ssd_tree_verify would run a pass of n nodes of the
 * model on this session under its current options: *path = 1 (one kernel
 * per sub-layer) or 2 (the persistent single launch).  Errors:
 * SSD_E_INVALID_ARG (null pointer, n outside [1, max_nodes]). */
ssd_status ssd_verify_path(const ssd_model *m, const ssd_kv *kv, int32_t n, int32_t *path);

/* Host-only: the persistent launch's work split for a model shape and a
 * count of 16-node tiles (1..4), as the session computes it.  tab receives
 * [256][32] int32 rows, one per compute workgroup (XCD x, rank r at row
 * 32 x + r): [0] the rank's position in the order its XCD's attention units
 * are dealt in (unit u goes to position u mod 32); [9] QKV row blocks, then
 * up to 4 row-block indices of W_qkv; [14] the same
 * for W_o; [19] for W_fc; [24] for W_pr; [29], [30] the workgroup's range of
 * LM-head row blocks.  xh[2x], xh[2x+1] bound XCD x's heads; xf[2x], xf[2x+1]
 * its hidden features in units of 32.  Errors: SSD_E_INVALID_ARG (null
 * pointer), SSD_E_UNSUPPORTED (the shape does not fit the split: head
 * dimension not 64, or too many units for a workgroup). */
ssd_status ssd_fused_plan(int32_t n_head, int32_t d_model, int32_t d_mlp, int32_t vocab, int32_t n_tiles,
                          int32_t *tab, int32_t *xh, int32_t *xf);

/* Stage timestamps of the persistent launch, for profiling.  With buf not
 * NULL, every later persistent pass of this session records for compute
 * workgroup g (XCD x, rank r: g = 32 x + r), layer l (n_layer + 1 rows; row
 * n_layer holds the final LayerNorm in stage 0 and the LM head in stage 1)
 * and stage s (8 per layer: LayerNorm, QKV, attention, out-projection,
 * LayerNorm, MLP up, MLP down, unused) three s_memrealtime readings (100 MHz):
 * stage entry, dependency met, stage published, at
 * buf[((g * (n_layer + 1) + l) * 8 + s) * 3 + k].  buf is caller-owned device
 * memory of 256 * (n_layer + 1) * 24 uint64 words for the largest model the
 * session runs; stages a workgroup skips keep old values.  NULL stops
 * recording.  Errors: SSD_E_INVALID_ARG (null session), SSD_E_UNSUPPORTED
 * (the session has no persistent pass). */
ssd_status ssd_kv_set_trace(ssd_kv *kv, uint64_t *buf);

/* The 8-bit copy of one weight matrix of a model from ssd_model_create_q8,
 * for checking: which = 0 W_qkv, 1 W_o, 2 W_fc, 3 W_pr (of `layer`), 4 the
 * LM head (layer ignored).  Writes codes[rows][cols] (int8, row-major as the
 * bfloat16 matrix) and scales[rows] (float32) to HOST memory; synchronises
 * the device.  Errors: SSD_E_INVALID_ARG (null pointer, bad id or layer, a
 * model without 8-bit weights), SSD_E_DEVICE. */
ssd_status ssd_model_q8_matrix(const ssd_model *m, int32_t which, int32_t layer, int8_t *codes, float *scales);

#ifdef __cplusplus
}
#endif
#endif
