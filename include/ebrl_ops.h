/*
 * ebrl_ops.h -- single-kernel entry points of the policy forward, exported
 * so each hot kernel can be checked and timed on its own.
 *
 * Same conventions as ebrl.h: device pointers, stream-ordered, status codes.
 */
#ifndef EBRL_OPS_H
#define EBRL_OPS_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* C[M, N] = A[M, K] * B[N, K]^T, the projection y = x W^T of every linear
 * layer (W stored [out, in]).  dtype EBRL_DTYPE_BF16: A and B bf16 (MFMA
 * path, fp32 accumulate); EBRL_DTYPE_FP32: float32.  C is float32 row-major
 * with leading dimension N.  Requires M, N >= 1, K >= 8 and K % 8 == 0;
 * the kernel choice (tile, split over K) depends only on (M, N, K).
 * stream: hipStream_t or NULL.  K splits (M < 256) write their partial sums
 * to a workspace the library allocates on the first call per (device,
 * stream) and keeps until the process ends, so calls on different streams
 * may overlap.  Returns EBRL_E_OOM if that allocation fails. */
int ebrl_op_gemm(int32_t dtype, const void* A, const void* B, float* C, int32_t M, int32_t N,
                 int32_t K, void* stream);

/* For callers that cannot allocate device memory: code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc.  The same
 * product as ebrl_op_gemm, bit for bit (same kernels and the same tile and
 * split choice), except that the partial sums and tile counters of a K split
 * live in a fixed device array of EBRL_OP_GEMM_NOALLOC_SCRATCH_BYTES that
 * each GPU the library runs on holds until the process ends; the call
 * allocates nothing and issues no memset.  Shapes whose split would write
 * more partial sums than the array holds return EBRL_E_INVALID (without a
 * split, e.g. M >= 256, any shape is accepted).  Every call on one GPU shares
 * that GPU's array: calls that overlap in time on one GPU (on different
 * streams or from different host threads) race and give wrong results;
 * calls ordered on one stream do not.  Same arguments and errors as
 * ebrl_op_gemm otherwise. */
#define EBRL_OP_GEMM_NOALLOC_SCRATCH_BYTES ((int64_t)16 * 1024 * 1024 + 4096 * 4)
int ebrl_op_gemm_noalloc(int32_t dtype, const void* A, const void* B, float* C, int32_t M, int32_t N,
                         int32_t K, void* stream);

/* Reads `bytes` of device memory at `buf` once with non-temporal 16-byte
 * loads (each workgroup a contiguous range).  Every loaded word feeds an XOR
 * that decides whether *out (device, 4 bytes) is written, so no load can be
 * dropped; *out is left unchanged unless that XOR equals 0x9E3779B9.  It is
 * the streaming-read reference for HBM-bound kernels: run on a CU-masked
 * stream it gives the bandwidth that share of the chip reaches.  Requires
 * bytes >= 16 and bytes % 16 == 0, buf and out non-NULL and buf 16-byte
 * aligned.  stream: hipStream_t or NULL.  Returns EBRL_E_INVALID on bad
 * arguments. */
int ebrl_op_stream_read(const void* buf, int64_t bytes, uint32_t* out, void* stream);

#ifdef __cplusplus
}
#endif
#endif /* EBRL_OPS_H */
