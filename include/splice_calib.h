/* splice_calib.h -- a plain HBM stream read, the measured ceiling that the
 * attention library's bandwidth is reported beside.
 *
 * Not part of the method: a measurement aid with no attention arithmetic.
 * The spliced decode attention reads each byte of its key/value caches once
 * per call, so the rate at which one kernel can stream bytes it reads once
 * from HBM bounds it more tightly than the 8 TB/s data-sheet figure.  This
 * library holds such a kernel: every work group reads one contiguous part of
 * a buffer with 16-byte non-temporal loads.
 *
 * Built by paper_2605_30574_amd/build.py into
 * paper_2605_30574_amd/libsplice_calib.so; it shares no code with the
 * attention library.
 */
#ifndef SPLICE_CALIB_H
#define SPLICE_CALIB_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SPLICE_CALIB_API __attribute__((visibility("default")))

#define SPLICE_CALIB_OK 0
#define SPLICE_CALIB_EINVAL (-1) /* a bad argument; nothing was launched */
#define SPLICE_CALIB_EHIP (-4)   /* the launch failed (hipGetLastError) */

/* Most work groups one call takes. */
#define SPLICE_CALIB_MAX_BLOCKS 65536

/* Read `bytes` bytes of device memory at `buf` once and write one 32-bit
 * word per work group to `sink`.
 *
 *   buf     device pointer, 16-byte aligned
 *   bytes   a positive multiple of 16; the 16-byte units are cut into
 *           `blocks` contiguous parts of ceil(units / blocks) units (the
 *           last parts may be shorter or empty), part b read by work group b
 *   sink    device memory of `blocks` 32-bit words: word b is the XOR of
 *           the four 32-bit words of every unit of part b (0 for an empty
 *           part), so the loads cannot be dropped and the result can be
 *           checked on the host
 *   blocks  work groups, 1 .. SPLICE_CALIB_MAX_BLOCKS
 *   stream  a hipStream_t, or NULL for the null stream
 *
 * Enqueues the kernel and returns; the caller owns every buffer and
 * synchronises.  Returns SPLICE_CALIB_OK, SPLICE_CALIB_EINVAL (NULL
 * pointers, misalignment, a size that is not a positive multiple of 16, or
 * a block count out of range; checked before anything is launched) or
 * SPLICE_CALIB_EHIP. */
SPLICE_CALIB_API int32_t splice_calib_stream_read(const void *buf, uint64_t bytes, uint32_t *sink,
                                                  int32_t blocks, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* SPLICE_CALIB_H */
