/*
 * samd_peaks.h - microbenchmarks of the MI355X (gfx950) ceilings that the SAMD
 * convolution kernels are measured against.  Library utilities for measurement; not
 * part of the convolution path.
 *
 * Each call enqueues one kernel on `stream` that performs a known amount of one kind of
 * work; the caller times it (HIP events) and divides samd_peak_work() by the time:
 *   SAMD_PEAK_MAD_I64_I32  exact signed 32x32 -> 64-bit multiply-adds (v_mad_i64_i32),
 *                          the SAMD multiply step; work = lane multiply-adds
 *   SAMD_PEAK_VALU_I32     full-rate 32-bit integer adds (v_add_u32); work = lane ops
 *   SAMD_PEAK_MFMA_I8      int8 matrix-core products (v_mfma_i32_16x16x64_i8), the
 *                          native 8-bit baseline's instruction; work = multiply-adds
 *   SAMD_PEAK_COPY         streaming copy of `bytes` bytes from src to dst (16-byte
 *                          loads and stores); work = bytes read + bytes written
 *   SAMD_PEAK_READ         streaming read of `bytes` bytes from src, one 4-byte sum per
 *                          workgroup written to dst; work = bytes read
 *   SAMD_PEAK_WRITE        streaming write of `bytes` bytes to dst (16-byte stores); work =
 *                          bytes written
 *   SAMD_PEAK_LDS          conflict-free 16-byte LDS reads (ds_read_b128), the int8
 *                          baseline's operand path; work = bytes read from LDS
 * Arguments:
 *   iters   loop trips of the compute and LDS kinds (1 .. 2^24; ignored by COPY and READ)
 *   blocks  workgroups of 256 threads (1 .. 2^20)
 *   src, dst COPY: device buffers of `bytes` bytes each (`bytes` a positive multiple of 16,
 *           both 16-byte aligned).  READ: src of `bytes` bytes (same rules), dst of
 *           `blocks` int32.  WRITE: dst of `bytes` bytes (same rules), src unused.  Compute kinds: src is unused and dst receives one int32 per
 *           thread (blocks * 256 values, so the work cannot be optimised away)
 * Returns SAMD_OK, SAMD_EINVAL for a bad argument, SAMD_EALIGN for a misaligned copy or
 * read buffer, or SAMD_EHIP for a launch error.
 */
#ifndef SAMD_PEAKS_H
#define SAMD_PEAKS_H

#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
    SAMD_PEAK_MAD_I64_I32 = 0,
    SAMD_PEAK_VALU_I32 = 1,
    SAMD_PEAK_MFMA_I8 = 2,
    SAMD_PEAK_COPY = 3,
    SAMD_PEAK_READ = 4,
    SAMD_PEAK_LDS = 5,
    SAMD_PEAK_WRITE = 6
};

int samd_peak_launch(int kind, int64_t iters, int32_t blocks, const void *src, void *dst, int64_t bytes,
                     hipStream_t stream);

/* Host-only: the work one samd_peak_launch with these arguments performs (see above). */
double samd_peak_work(int kind, int64_t iters, int32_t blocks, int64_t bytes);

#ifdef __cplusplus
}
#endif

#endif /* SAMD_PEAKS_H */
