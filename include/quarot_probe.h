/*
 * libquarot_probe: measurement utilities beside libquarot (not steps of the
 * method, and not part of libquarot itself).  They give the attainable rate
 * of the GEMMs' matrix instructions under load and the device's peak clock,
 * against which the benchmark reads the GEMMs' achieved rates besides the
 * published peaks.  Status codes as in quarot.h; arguments are checked on
 * the host before any device work, and on error nothing is written.
 *
 * quarot_device_peaks: the current device's compute-unit count and peak
 * shader clock in kHz (hipDeviceGetAttribute), from which the int8 MFMA
 * peak is CUs x clock x 8192 ops per clock per CU.  QUAROT_ERR_NO_DEVICE
 * unless the current device is a gfx950.
 *
 * quarot_mfma_probe: enqueues blocks x 512 threads (8 waves per block, two
 * per SIMD) whose waves run iters x 32 v_mfma_i32_16x16x64_i8 each on
 * changing operands: blocks x 8 x iters x 32 x 16384 multiply-adds in all;
 * out: int32 [blocks * 512], written (a checksum of no meaning), 16-byte
 * aligned device memory owned by the caller.  The caller times it on its
 * stream (a hipStream_t, or NULL for the default stream);
 * 1 <= blocks, iters <= 2^20.
 *
 * quarot_mfma_probe_fp6: the same with v_mfma_f32_16x16x128_f8f6f4 on e3m2
 * operands (the instruction of quarot_w4a4_gemm_e3m2): blocks x 8 x iters
 * x 32 x 32768 multiply-adds.
 *
 * quarot_probe_last_hip_error: the hipError_t behind this thread's last
 * QUAROT_ERR_HIP from these calls.
 */
#ifndef QUAROT_PROBE_H
#define QUAROT_PROBE_H

#include "quarot.h"

#ifdef __cplusplus
extern "C" {
#endif

quarot_status quarot_device_peaks(int *cu_count, int *max_clock_khz);
quarot_status quarot_mfma_probe(int32_t *out, int64_t blocks, int iters, void *stream);
quarot_status quarot_mfma_probe_fp6(int32_t *out, int64_t blocks, int iters, void *stream);
int quarot_probe_last_hip_error(void);

#ifdef __cplusplus
}
#endif

#endif
