/*
 * qwam_probe.h -- measurement probes of libqwam (MI355X, gfx950).
 *
 * Not part of the ASP layer.  They measure what the chip itself sustains, so
 * that the benchmark can put each kernel's rate beside a measured ceiling as
 * well as beside the vendor figure: a matrix-core loop per MFMA format, a
 * float32 VALU loop, a streaming copy and an empty kernel.  Each call only
 * enqueues its kernel on `stream` (a hipStream_t; NULL = the null stream);
 * time it with events on that stream.  Arguments are checked on the host
 * before any HIP call; on error nothing is enqueued and
 * qwam_probe_last_error() describes the failure.
 */
#ifndef QWAM_PROBE_H
#define QWAM_PROBE_H

#include <stdint.h>

#include "qwam.h"

#ifdef __cplusplus
extern "C" {
#endif

/* matrix-core formats of qwam_probe_mfma; the work per instruction is
 * 2 * 32 * 32 * K operations, K given after each name */
#define QWAM_PROBE_MFMA_FP6 0     /* v_mfma_scale_f32_32x32x64_f8f6f4, FP6 e2m3 operands, K = 64 */
#define QWAM_PROBE_MFMA_FP8 1     /* the same instruction with FP8 e4m3 operands, K = 64          */
#define QWAM_PROBE_MFMA_FP4 2     /* the same instruction with FP4 e2m1 operands, K = 64          */
#define QWAM_PROBE_MFMA_I8 3      /* v_mfma_i32_32x32x32_i8, K = 32                               */
#define QWAM_PROBE_MFMA_BF16 4    /* v_mfma_f32_32x32x16_bf16, K = 16                             */
#define QWAM_PROBE_MFMA_BF16_2B 5 /* v_mfma_f32_32x32x4_2b_bf16: two 32 x 32 blocks, K = 4 each    */

/*
 * `workgroups` workgroups of 256 threads (4 waves); every wave issues
 * 4 * iters MFMAs of format `kind` (four independent accumulators).
 * out: device float [workgroups * 256], written (keeps the work alive).
 * Operations performed: workgroups * 4 * 4 * iters * 2 * 32 * 32 * K
 * (times 2 blocks for QWAM_PROBE_MFMA_BF16_2B).
 */
qwam_status qwam_probe_mfma(int32_t kind, int32_t workgroups, int32_t iters, float *out, void *stream);

/*
 * `workgroups` workgroups of 256 threads; every thread runs 256 * iters
 * float32 fused multiply-adds in 16 independent chains (non-packed VALU
 * instructions).  Flops performed: workgroups * 256 * 256 * iters * 2.
 * out: device float [workgroups * 256], written.
 */
qwam_status qwam_probe_valu_fma(int32_t workgroups, int32_t iters, float *out, void *stream);

/*
 * dst[0 .. bytes) = src[0 .. bytes), 16 bytes per lane and access,
 * grid-stride over `workgroups` workgroups of 256 threads.  bytes % 16 == 0,
 * both buffers 16-byte aligned and disjoint.  HBM bytes moved: 2 * bytes.
 */
qwam_status qwam_probe_copy(const void *src, void *dst, int64_t bytes, int32_t workgroups, void *stream);

/* One workgroup of 64 threads that does nothing: the launch floor. */
qwam_status qwam_probe_empty(void *stream);

/* Message of the calling thread's last failing probe call ("" if none). */
const char *qwam_probe_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* QWAM_PROBE_H */
