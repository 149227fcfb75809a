/*
 * hbm_probe.h - C ABI of libhbm_probe.so: streaming kernels that measure the
 * practical HBM ceiling for the read/write mix of RRQ package construction.
 * Construction reads 2 bytes per weight (bfloat16) and writes 1.25 (four
 * 2-bit code planes plus binary32 scale and zero per group of 128), so the
 * mixed probe reads B bytes and writes 5B/8 bytes with the same kind of wide,
 * coalesced accesses, and no arithmetic; the read-only and write-only probes
 * give each direction's own ceiling, and the construct-pattern and
 * reconstruct-pattern probes replay those kernels' own loads and stores; two
 * machine probes time instruction issue (matrix-core and vector) and LDS
 * reads. Measurement aids only: they compute nothing of the method.
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

/*
 * hbm_probe_construct - enqueue one pass with package construction's own
 * memory traffic and no quantization arithmetic: n_groups groups of
 * group_size bfloat16 weights are read once, in the construct kernel's tiles
 * of 64 groups (one wave each, next tile prefetched, LDS transpose), and per
 * stage each group stores its group_size / 16 code words, one 32-bit scale
 * and one 32-bit zero-point into the planes of rrq_construct's layout. With
 * w[0..group_size/2 - 1] the group's 32-bit words (little-endian pairs of
 * bfloat16) and k the stage:
 *   codes[k][g * group_size/16 + j] = (XOR of w[j + m * group_size/16] over m) ^ k
 *   scales[k][g] = w[0] ^ k,   zeros[k][g] = w[1] ^ k.
 *
 *   W            device, n_groups * group_size * 2 bytes, 16-byte aligned.
 *   n_groups     >= 1.
 *   group_size   32, 64 or 128.
 *   n_stages     1 .. 4.
 *   codes        device, n_stages * n_groups * group_size / 16 uint32, 16-byte aligned.
 *   scales,
 *   zeros        device, n_stages * n_groups uint32 each, 4-byte aligned.
 *   blocks_per_cu  resident one-wave workgroups per compute unit, 1 .. 32;
 *                0 = the construct kernel's 8.
 *
 * Returns 0, or 1 (NULL), 2 (misaligned), 3 (bad size or argument) with
 * nothing enqueued, or 7 if the launch failed. Outputs must not overlap W or
 * each other. The caller owns every buffer; nothing is allocated.
 */
int hbm_probe_construct(const void *W, int64_t n_groups, int32_t group_size, int32_t n_stages,
                        uint32_t *codes, uint32_t *scales, uint32_t *zeros,
                        int32_t blocks_per_cu, hipStream_t stream);

/*
 * hbm_probe_reconstruct - enqueue one pass with the memory traffic of
 * rrq_reconstruct (k_stages prefix, bfloat16 output) and no dequantization
 * arithmetic: for every chunk of 8 consecutive elements (16 output bytes)
 * and every stage t < k_stages it loads the chunk's code word (word
 * e / 16 of plane t), its group's scale and its group's zero-point (32-bit
 * words of plane t), and stores the chunk once. With x the XOR over the
 * stages of those three words, chunk c (elements 8c .. 8c + 7) stores the
 * 32-bit words x, x + 1, x + 2, x + 3 at out + 4c.
 *
 *   codes       device, planes of n_groups * group_size / 16 uint32 (at least
 *               k_stages planes), 16-byte aligned.
 *   scales,
 *   zeros       device, planes of n_groups uint32 each, 4-byte aligned.
 *   n_groups    >= 1.
 *   group_size  32, 64 or 128.
 *   k_stages    1 .. 4.
 *   out         device, n_groups * group_size * 2 bytes, 16-byte aligned.
 *   blocks_per_cu  resident 256-thread workgroups per compute unit, 1 .. 32;
 *               0 = the reconstruct kernel's 2.
 *
 * Returns as hbm_probe_construct.
 */
int hbm_probe_reconstruct(const uint32_t *codes, const uint32_t *scales, const uint32_t *zeros,
                          int64_t n_groups, int32_t group_size, int32_t k_stages, uint32_t *out,
                          int32_t blocks_per_cu, hipStream_t stream);

/*
 * hbm_probe_issue - machine probe of instruction issue: one 4-wave workgroup
 * per compute unit and waves_per_simd (one wave per SIMD each); every wave
 * runs iters iterations of, by mode, 0: 16 v_mfma_f32_16x16x32_bf16 on 4
 * accumulator chains; 1: 64 binary32 FMAs on 8 chains; 2: both. Each wave
 * writes the s_memtime ticks of its loop to ticks[wave] (global wave index),
 * each thread a checksum to out (so that no work is folded away).
 *
 *   out        device, out_len floats, >= CUs x waves_per_simd x 256.
 *   ticks      device, ticks_len int64, >= CUs x waves_per_simd x 4.
 *   waves_per_simd  1 .. 4; iters >= 1.
 *
 * Returns 0, 1 (NULL), 3 (bad argument or size) with nothing enqueued, or 7.
 */
int hbm_probe_issue(int mode, int waves_per_simd, int iters, float *out, size_t out_len,
                    long long *ticks, size_t ticks_len, hipStream_t stream);

/*
 * hbm_probe_lds - machine probe of LDS reads: one workgroup of
 * waves_per_cu (4 or 8) waves per compute unit on a 96 KiB LDS array; every
 * wave runs iters iterations of 16 reads of 16 bytes per lane (a wave's
 * 64 slots distinct) and writes the s_memtime ticks of its loop to
 * ticks[wave], each thread a checksum to out.
 *
 *   out        device, out_len uint32, >= CUs x waves_per_cu x 64.
 *   ticks      device, ticks_len int64, >= CUs x waves_per_cu.
 *
 * Returns as hbm_probe_issue.
 */
int hbm_probe_lds(int waves_per_cu, int iters, uint32_t *out, size_t out_len, long long *ticks,
                  size_t ticks_len, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* HBM_PROBE_H */
