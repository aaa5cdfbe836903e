/*
 * instantmimic_calib.h -- measurement probes of the GPU itself.
 *
 * Not part of the method: these entry points run micro-kernels whose timings
 * tell what the MI355X sustains for the instruction mixes the library's own
 * kernels use (MFMA chains, LDS fragment reads, streaming global reads), so
 * that the library kernels' fractions of the published peaks can be read
 * against what is reachable.  They live in libinstantmimic.so next to the
 * method's entry points and share its status codes.
 *
 * Each call only enqueues one kernel on `stream` (a hipStream_t, or NULL for
 * the null stream) and returns; the caller times it (HIP events on the same
 * stream) and synchronises.  All pointers are device pointers owned by the
 * caller.  Arguments are checked before anything is launched: a bad one
 * returns IM_ERR_INVALID_ARG with nothing enqueued; a failed launch returns
 * IM_ERR_HIP.
 */
#ifndef INSTANTMIMIC_CALIB_H
#define INSTANTMIMIC_CALIB_H

#include "instantmimic.h"

#ifdef __cplusplus
extern "C" {
#endif

enum {
    IM_CALIB_MFMA_BF16 = 0,   /* v_mfma_f32_32x32x16_bf16: 32768 flop per instruction */
    IM_CALIB_MFMA_F32 = 1     /* v_mfma_f32_32x32x2_f32:   4096 flop per instruction */
};

/* MFMA throughput.  `blocks` blocks of 256 threads (4 wavefronts); every
 * wavefront runs `iters` rounds of 8 independent MFMAs of the given kind on
 * register operands.  Work = 4 * blocks * iters * 8 * (flop per instruction).
 * out: float[256 * blocks], one checksum per thread (keeps the work live). */
im_status im_calib_mfma(int kind, int64_t iters, int blocks, float *out, void *stream);

/* LDS read throughput.  `blocks` blocks of 64 * waves threads (waves in
 * 1..16), one 64 KB LDS array each; every wavefront runs `iters` rounds of 16
 * reads of `width` bytes per lane (16: ds_read_b128 in the GEMM's fragment
 * pattern, 128-byte rows with 16-byte chunks XOR-swizzled by (row / 2) % 8;
 * 8: ds_read_b64 of consecutive 8-byte words) and waits for them.  Bytes read
 * per block = waves * 64 * width * 16 * iters.
 * out: uint32[64 * waves * blocks], one checksum per thread. */
im_status im_calib_lds(int width, int waves, int64_t iters, int blocks, uint32_t *out, void *stream);

/* Streaming global read.  `blocks` blocks of 256 threads read the `bytes`
 * bytes at src (16-byte aligned, a multiple of 16) in 16-byte words, thread t
 * of the grid taking words t, t + 256 * blocks, ..., `passes` times over.
 * Bytes read = passes * bytes.  out: uint32[256 * blocks], one checksum per
 * thread. */
im_status im_calib_read(const void *src, int64_t bytes, int passes, int blocks, uint32_t *out,
                        void *stream);

#ifdef __cplusplus
}
#endif

#endif /* INSTANTMIMIC_CALIB_H */
