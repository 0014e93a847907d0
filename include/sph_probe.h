/*
 * sph_probe.h - measurement helpers of libsph (not steps of the method).
 *
 * They give the attainable rates a projection kernel is compared with,
 * measured on the device itself with kernels of the same kind:
 *
 *   sph_probe_read  streams a buffer once with 16-byte non-temporal loads,
 *                   the access the skinny projection makes of its weight
 *                   rows: attainable HBM read bandwidth.
 *   sph_probe_mfma  a loop of independent v_mfma_f32_32x32x16_bf16 on
 *                   random bf16 operands that change every iteration:
 *                   attainable dense bf16 matrix-core rate.
 *
 * Both only enqueue one kernel on `stream` (a hipStream_t, NULL = default)
 * and return; the caller times it (for example with events on the same
 * stream).  A negative return value is an error (the codes of sph.h);
 * nothing has been enqueued and sph_last_error() has the message.
 */
#ifndef SPH_PROBE_H
#define SPH_PROBE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Read `bytes` bytes of device memory at `buf` once.  `buf` must be 16-byte
 * aligned and `bytes` a positive multiple of 16.  `sink` is one device
 * float the kernel may write (so the loads cannot be dropped). */
int sph_probe_read(const void* buf, int64_t bytes, float* sink, void* stream);

/* Launch one MFMA loop of `iters` iterations (1 <= iters <= 2^30): 256
 * workgroups of 4 waves, each wave issuing 32 MFMAs per iteration.  The
 * launch's floating-point operations are stored in *flops_out (host).
 * `sink` is one device float the kernel may write. */
int sph_probe_mfma(int64_t iters, float* sink, void* stream, double* flops_out);

#ifdef __cplusplus
}
#endif

#endif /* SPH_PROBE_H */
