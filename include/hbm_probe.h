/*
 * hbm_probe.h - C ABI of libhbm_probe.so: streaming kernels that measure the
 * practical HBM ceiling for the read/write mix of RRQ package construction.
 * Construction reads 2 bytes per weight (bfloat16) and writes 1.25 (four
 * 2-bit code planes plus binary32 scale and zero per group of 128), so the
 * mixed probe reads B bytes and writes 5B/8 bytes with the same kind of wide,
 * coalesced accesses, and no arithmetic; the read-only and write-only probes
 * give each direction's own ceiling. Measurement aids only: they compute
 * nothing of the method.
 */
#ifndef HBM_PROBE_H
#define HBM_PROBE_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/*
 * hbm_probe_stream - enqueue one pass: src is read in full; of every 128
 * bytes of src, the first 80 are written to the next 80 bytes of dst.
 *
 *   src        device, src_bytes bytes, 16-byte aligned (read only).
 *   src_bytes  a positive multiple of 128.
 *   dst        device, src_bytes / 8 * 5 bytes, 16-byte aligned (written);
 *              must not overlap src.
 *   stream     HIP stream the work is enqueued on.
 *
 * Returns 0, or 1 (NULL pointer), 2 (misaligned pointer), 3 (bad size) with
 * nothing enqueued, or 7 if the launch failed. The caller owns both buffers;
 * the library allocates nothing.
 */
int hbm_probe_stream(const void *src, size_t src_bytes, void *dst, hipStream_t stream);

/*
 * hbm_probe_read - enqueue one pass that reads all of src (nontemporal 16-byte
 * loads) and XORs the XOR of all its 32-bit words into *out (the caller sets
 * *out beforehand, e.g. to 0).
 *
 *   src        device, src_bytes bytes, 16-byte aligned (read only).
 *   src_bytes  a positive multiple of 16.
 *   out        device, one uint32_t, 4-byte aligned (read and written).
 *
 * Returns 0, 1 (NULL), 2 (misaligned), 3 (bad size) with nothing enqueued,
 * or 7 if the launch failed.
 */
int hbm_probe_read(const void *src, size_t src_bytes, uint32_t *out, hipStream_t stream);

/*
 * hbm_probe_write - enqueue one pass that writes value into every 32-bit word
 * of dst (16-byte stores, one workgroup per compute unit).
 *
 *   dst        device, dst_bytes bytes, 16-byte aligned (written).
 *   dst_bytes  a positive multiple of 16.
 *
 * Returns as hbm_probe_read.
 */
int hbm_probe_write(void *dst, size_t dst_bytes, uint32_t value, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* HBM_PROBE_H */
