/* Achievable-peak calibration of the device (measurement support, not part of the
 * KV-sharing method).
 *
 * The datasheet peaks of an MI355X (bf16 dense matrix cores 2516.6 TFLOP/s at the 2.4 GHz
 * boost clock, HBM3E 8 TB/s) are not what a kernel can reach: under sustained matrix load
 * with operands that change every instruction the part runs below its boost clock, and
 * streaming reads top out below the HBM interface rate.  These two kernels measure both
 * ceilings on the device at hand so that a roofline fraction can be stated against the
 * datasheet and against what the device delivers.  Both run on libkvpipe.so and are
 * exported beside the method's entry points.
 *
 * Errors: KVP_E_INVALID_ARG for a bad argument, KVP_E_HIP for a failed launch (message in
 * kvp_last_error()).  Calls are asynchronous on `stream` (a hipStream_t, NULL = default);
 * the caller times them with events on that stream.
 */
#ifndef KVP_CALIB_H_
#define KVP_CALIB_H_

#include <stddef.h>

#ifdef __cplusplus
extern "C" {
#endif

/* bf16 matrix-core loop: one workgroup of 8 waves per compute unit (two per SIMD); every
 * wave issues `iters` x 16 v_mfma_f32_32x32x16_bf16 with four independent accumulators
 * and sixteen registers of pseudo-random bf16 values (magnitudes 2^-3 .. 2^1) combined so
 * that consecutive instructions read different data.  iters even, in [2, 2^24].  sink:
 * device buffer of at least 4 bytes, written only if the accumulators hit an impossible
 * value (keeps the work alive).  *flops receives the floating-point operations of the
 * launch (2 * 32 * 32 * 16 per instruction). */
int kvp_calib_mfma_bf16(int iters, void* sink, double* flops, void* stream);

/* Streaming HBM read of `bytes` bytes at device address src (16-byte aligned; bytes a
 * positive multiple of 65536) by 64 waves per compute unit, each streaming a contiguous
 * share in 8 KB blocks of eight 1 KB wave-loads (16 bytes per lane), all eight in flight.
 * sink: device buffer of at least 16 bytes, written only if the xor of all data hits an
 * impossible value.  The caller provides a buffer much larger than the 256 MB last-level
 * cache, so the reads come from HBM. */
int kvp_calib_stream_read(const void* src, size_t bytes, void* sink, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* KVP_CALIB_H_ */
