/* Measured device ceilings: libxmix_ceiling.so.
 *
 * Two measurement aids that sit beside the hook-step library.  They are not
 * steps of the method and no hook-step call uses them.  They show what the
 * GPU at hand really reaches, so that the encode kernels' rates can be read
 * against measured ceilings as well as the published peaks (MI355X: HBM
 * 8 TB/s, dense bf16 MFMA 2.5 PFLOP/s).
 *
 * Both calls are asynchronous on `stream` (a hipStream_t; NULL is the null
 * stream) and allocate nothing.  Time them with events around the launch.
 * They return 0 on success, 1 for an invalid argument (nothing launched) and
 * 4 when the launch fails.
 */
#ifndef XMIX_CEILING_H
#define XMIX_CEILING_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Reads `bytes` bytes of device memory at `buf` once, with 16-byte
 * nontemporal loads, two workgroups of 256 threads per compute unit; in each
 * round the grid reads one contiguous span.  `buf` is a device pointer,
 * 16-byte aligned, `bytes` a non-zero multiple of 16.  `sink` is a device
 * word that the kernel never changes for real data (it only keeps the
 * compiler from dropping the loads).  Pass a buffer larger than the 256 MB
 * infinity cache, or rotate between several, to time HBM rather than cache. */
int xmix_ceiling_read(const void* buf, uint64_t bytes, uint32_t* sink, void* stream);

/* One workgroup of four waves per compute unit; each wave runs `iters`
 * rounds of eight independent 32x32x16 bf16 MFMAs with register operands
 * and fp32 accumulation.  `sink` is a device float the kernel never writes
 * for these operands.  `*flops` (host, may be NULL) receives the launch's
 * dense flop count, 2 * 32 * 32 * 16 per MFMA. */
int xmix_ceiling_mfma(int32_t iters, float* sink, double* flops, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* XMIX_CEILING_H */
