/*
 * pipeboost_ops.h -- kernel-level entry points of libpipeboost.so.
 *
 * Each call runs one kernel of the prefill (plus its split-K reduce where the
 * launcher splits) on caller-provided device buffers, on the given stream,
 * asynchronously.  They exist to test every kernel against the CPU oracle's
 * component functions and to time kernels in isolation; the model API in
 * pipeboost.h is the product path.  All pointers are device pointers, all
 * matrices row-major with the reduction dimension contiguous; "dt" is
 * bfloat16 (dtype 0) or IEEE binary16 (dtype 1).  Every call returns a
 * pb_status (PB_EINVAL for unsupported shapes, PB_EHIP for launch failures,
 * message in pb_last_error()).
 */
#ifndef PIPEBOOST_OPS_H
#define PIPEBOOST_OPS_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Projection GEMM Y = X W^T (fp32 accumulate) with an epilogue
 * (Section 2.1: the decoder's linear layers; bias as in OPT):
 *   epi 0: C = dt((Y + bias) * (n < qcols ? qscale : 1))   (q, k, v projection)
 *   epi 1: C = dt(max(Y + bias, 0))                        (fc1 with ReLU)
 *   epi 2: R += Y + bias, R fp32 [M, N] (ldr = N)           (o and fc2, residual)
 * X [M, K] dt, W [N, K] dt, bias [N] dt, C [M, N] dt (ldc = N).  Requires
 * N % 64 == 0 and K % 64 == 0.  workspace (fp32 scratch for split-K partials,
 * may be NULL) of workspace_bytes. */
int pb_op_gemm(int32_t dtype, int32_t epi, const void* X, const void* W, const void* bias,
               void* C, float* R, int32_t M, int32_t N, int32_t K, float qscale, int32_t qcols,
               void* workspace, size_t workspace_bytes, void* stream);

/* pb_op_gemm with the unmerged LoRA expand folded into the same accumulation
 * as extra K tiles (Section 2.1: the adapter adds s (x A) B on top of the
 * fixed W; Section 4.2.2: sequences of one batch may use different adapters):
 *   Y[m, n] = X[m] . W[n] + Z[m, g zs .. g zs + K2) . W2[n]   if bit g of group_mask
 *           = X[m] . W[n]                                     otherwise,
 * with g = n / group (the output group: q, k, v of a fused projection),
 * then the epilogue of pb_op_gemm.  Z [M, ldz] dt holds each row's scaled
 * shrink s (x A_slot) in its adapter slot's columns of every group block
 * (zeros in the other slots' columns, so rows of different adapters, or none,
 * share the launch); W2 [N, K2] dt holds the B matrices of all slots side by
 * side.  K2 % 64 == 0, group % 64 == 0; other requirements and the workspace
 * as pb_op_gemm. */
int pb_op_gemm_lora(int32_t dtype, int32_t epi, const void* X, const void* W, const void* bias, void* C,
                    float* R, int32_t M, int32_t N, int32_t K, const void* Z, int32_t ldz, int32_t zs,
                    const void* W2, int32_t K2, int32_t group, uint32_t group_mask, float qscale,
                    int32_t qcols, void* workspace, size_t workspace_bytes, void* stream);

/* pb_op_gemm for callers that cannot allocate (code under HIP graph capture,
 * tight serving loops, harnesses that forbid hipMalloc): the same operands,
 * epilogues and kernels, with the split-K partials in a 64 MiB device array
 * of the library instead of a caller workspace.  The call allocates nothing
 * (no hipMalloc, hipFree or allocating library routine); the array is part
 * of the library's code object, one copy per GPU, held until the process
 * ends.  The result is bit-identical to pb_op_gemm given a 64 MiB workspace.
 * Products are limited to M * N * 4 <= 64 MiB (PB_EINVAL above it: use
 * pb_op_gemm).  The array of the current device is used, so `stream` must
 * belong to that device.  Every call on a GPU shares that GPU's array: calls
 * that overlap on one GPU (other streams or threads) race. */
int pb_op_gemm_noalloc(int32_t dtype, int32_t epi, const void* X, const void* W, const void* bias,
                       void* C, float* R, int32_t M, int32_t N, int32_t K, float qscale,
                       int32_t qcols, void* stream);

/* Causal multi-head self-attention over B sequences of T tokens (Section 2.1:
 * prefill self-attention; token j attends to tokens 0..j).  qkv [B*T, 3*H*hd]
 * dt with q already divided by sqrt(hd), out [B*T, H*hd] dt; hd in {64, 128}. */
int pb_op_attention(int32_t dtype, const void* qkv, void* out, int32_t B, int32_t T,
                    int32_t H, int32_t hd, void* stream);

/* LayerNorm of rows of an fp32 matrix x [rows, d]: out = LN(x) * g + b with
 * fp32 statistics (biased variance); g, b [d] dt; out [rows, d] dt, or fp32
 * when out_f32 != 0.  d % 4 == 0, d <= 16384. */
int pb_op_layernorm(int32_t dtype, const float* x, const void* g, const void* b, void* out,
                    int32_t out_f32, int32_t rows, int32_t d, float eps, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* PIPEBOOST_OPS_H */
