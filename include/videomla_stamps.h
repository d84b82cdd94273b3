/* Phase stamps: the diagnostic build of the library.
 *
 * libvideomla_stamps.so is built from the same sources as libvideomla.so, with
 * VMLA_PHASE_STAMPS defined. It exports every call of videomla.h, with the same behaviour and
 * results, plus videomla_stamps_attach below. Its kernels record, at named points of each
 * workgroup's life, the GPU's 100 MHz real-time counter. The points are the ones that show
 * where a kernel's time goes: operands landed, contraction done, epilogue, stores complete.
 * The records go into a caller-owned device buffer. The stores and waits add a little time
 * to each stamped kernel. In libvideomla.so the stamp points compile to nothing, and it does
 * not export this call.
 *
 * It is for measurement, not for serving. The stamped kernels are these steps of the method:
 * - the cache write (compression and key RoPE, Eqs. 1 and 5);
 * - the query absorption (Eq. 8);
 * - the latent attention (Eqs. 7 and 10);
 * - the merge of key splits with the value up-projection W_UV (Eq. 2).
 */
#ifndef VIDEOMLA_STAMPS_H
#define VIDEOMLA_STAMPS_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Buffer layout: uint64 [kernel][workgroup][wave][point], sizes below. Entry (k, w, v, p) is
 * the counter value at which wave v of workgroup w of the last launch of kernel k reached
 * point p. The workgroup index is blockIdx.x + gridDim.x (blockIdx.y + gridDim.y blockIdx.z).
 * A launch writes only the entries it reaches, so the caller zeroes the buffer before the
 * call it wants to read. Workgroups at or past 2048 and waves at or past 8 are not recorded.
 *
 * Kernels and points:
 * - 0, the cache write with packed weights, up to 32 tokens per compute unit:
 *   0 start; 1 the first half of x landed (the angle tables are done too);
 *   2 the second half landed; 3 last MFMA issued;
 *   4 sums of squares exchanged; 5 output tile complete; 6 stores complete.
 * - 1, the cache write with packed weights, more than 32 tokens per compute unit. Compute
 *   waves 0..6:
 *   0 start; 1 tables done; 2 + p phase p of x landed (p < 10);
 *   12 last MFMA issued; 13 sums of squares exchanged; 14 output tile complete;
 *   15 stores complete.
 *   The loader wave (the last one) records 0 and 15 only.
 * - 2, the query absorption:
 *   0 start; 1 W_UK_h staged in LDS; 2 last MFMA issued (1 and 2 of the first pass over
 *   W_UK_h's columns, the only one up to d_c = 192); 3 latent part written;
 *   4 RoPE part written; 5 rows staged; 6 stores complete.
 * - 3, the latent attention (latent form only; the dense and materialized kernels record
 *   nothing):
 *   0 start; 1 first two tiles landed;
 *   2 + 2i / 3 + 2i the instruction stream of the workgroup's step 200 + i ended / its
 *   barrier passed (i < 4). The stream's end is read before the step's wait for its tile
 *   loads, and stored only after the barrier, so the wait has no stamp store to drain;
 *   10 last step done; 11 partial results stored;
 *   12 the first segment's last step done and 13 its partial results issued (every
 *   workgroup); 14 the second segment's first two tiles landed (workgroups with a second
 *   segment only).
 * - 4, the merge of key splits with W_UV_h:
 *   0 start; 1 coefficients and W_UV_h in LDS; 2 merged o_lat tile complete;
 *   3 last MFMA issued; 4 output rows staged; 5 stores complete.
 */
#define VIDEOMLA_STAMP_KERNELS 5
#define VIDEOMLA_STAMP_WORKGROUPS 2048
#define VIDEOMLA_STAMP_WAVES 8
#define VIDEOMLA_STAMP_POINTS 16
#define VIDEOMLA_STAMP_BUFFER_BYTES \
  ((int64_t)VIDEOMLA_STAMP_KERNELS * VIDEOMLA_STAMP_WORKGROUPS * VIDEOMLA_STAMP_WAVES * VIDEOMLA_STAMP_POINTS * 8)

/* Sets the buffer that the launches of every later call record into.
 * - device_buffer: device memory of at least VIDEOMLA_STAMP_BUFFER_BYTES bytes, 8-byte
 *   aligned, owned by the caller. The caller keeps it alive while such calls run. NULL
 *   detaches the buffer, and later calls record nothing.
 * - The setting is one process-wide pointer in the diagnostic build.
 * Errors: VIDEOMLA_EINVAL if bytes is below VIDEOMLA_STAMP_BUFFER_BYTES for a non-NULL
 * buffer; VIDEOMLA_EALIGN if the buffer is not 8-byte aligned. */
int videomla_stamps_attach(void* device_buffer, int64_t bytes);

#ifdef __cplusplus
}
#endif

#endif /* VIDEOMLA_STAMPS_H */
