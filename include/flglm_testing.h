/*
 * flglm_testing.h - single-kernel entry points of the FL-GLM server-stack
 * library, exported for per-kernel parity tests.  Not part of the product
 * ABI (flglm.h); same conventions: 0 or a negative FL_ERR_* code,
 * fl_last_error() for the message, device pointers 16-byte aligned, leading
 * dimensions multiples of 8 elements, `stream` a hipStream_t.
 *
 * dtype: FL_BF16 or FL_F32 (element type of every non-fp32 buffer).
 */
#ifndef FLGLM_TESTING_H_
#define FLGLM_TESTING_H_

#include <stdint.h>

#include "flglm.h"

#ifdef __cplusplus
extern "C" {
#endif

#define FL_GEMM_NT 0 /* C[m,n] = sum_k A[m*lda+k] B[n*ldb+k]   (forward linear)       */
#define FL_GEMM_NN 1 /* C[m,n] = sum_k A[m*lda+k] B[k*ldb+n]   (input gradient)       */
#define FL_GEMM_TN 2 /* C[m,n] = sum_k A[k*lda+m] B[k*ldb+n]   (weight gradient)      */

#define FL_EPI_STORE 0     /* C = acc                                   */
#define FL_EPI_BIAS 1      /* C = acc + bias[n]                         */
#define FL_EPI_BIAS_RES 2  /* C = acc + bias[n] + R[m*ldr+n]            */
#define FL_EPI_BIAS_GELU 3 /* C = z = acc + bias[n]; C2 = gelu_tanh(z)  */
#define FL_EPI_GELU_BWD 4  /* C = acc * gelu_tanh'(Z[m*ldz+n])          */
#define FL_EPI_ACC_F32 5   /* C (fp32) += acc                           */
#define FL_EPI_RES 6       /* C = acc + res_scale * R[m*ldr+n]          */

/* Matrix-core GEMM as used by the linear layers.  Supported pairs: NT with
 * STORE/BIAS/BIAS_RES/BIAS_GELU, NN with STORE/GELU_BWD/RES, TN with ACC_F32.
 * res_scale multiplies R in BIAS_RES and RES (1: plain residual).
 * part / part_bytes: optional device fp32 scratch (16-byte aligned) that
 * lets the bf16 kernel split the reduction of a last, partial round of
 * tiles over more compute units (NULL / 0: never split).
 * b_rows > 0: B holds only that many rows (its N index for NT, its
 * reduction index for NN and TN); the rest read as zero and are never
 * touched (0: B is complete).
 * colsum (NULL: none): for bf16 NN GELU_BWD on the LDS-DMA kernel only
 * (FL_ERR_ARG otherwise), device fp32 [ceil(M/256)][N] that receives, per
 * 256-row block, the column sums of the stored C (the partial layout of the
 * bias-gradient column sums).
 * Requirements: N % 128 == 0 (bf16) or N % 64 == 0 (fp32); K % 64 == 0 for
 * NT and NN; M % 8 == 0 for TN. */
int fl_test_gemm(int dtype, int layout, int epi, const void* A, const void* B, void* C, int M, int N, int K,
                 int64_t lda, int64_t ldb, int64_t ldc, const void* bias, const void* R, int64_t ldr, void* C2,
                 int64_t ldc2, const void* Z, int64_t ldz, float* part, int64_t part_bytes, int b_rows,
                 float res_scale, float* colsum, void* stream);

/* LayerNorm over rows of x [T, H] (H % 256 == 0, H <= 4096). */
int fl_test_layernorm_fwd(int dtype, const void* x, const void* g, const void* b, void* y, float* mean, float* rstd,
                          int T, int H, float eps, void* stream);
/* dx = dres + LayerNorm input gradient of dy (the LN gain/shift gradients
 * are produced by the column-sum kernel, see fl_test_colsum). */
int fl_test_layernorm_bwd(int dtype, const void* dy, const void* x, const float* mean, const float* rstd,
                          const void* g, const void* dres, void* dx, int T, int H, void* stream);
/* The LayerNorm backward the stack runs, fused with its column sums: dx as
 * above (dres may be NULL: no residual), and, when given (fp32, +=),
 * dgamma[n] = sum_t dy[t][n] xh[t][n], dbeta[n] = sum_t dy[t][n] (both or
 * neither) and dsum[n] = sum_t dx[t][n] (the stored, rounded dx).  partial:
 * device fp32 scratch of 3 * 512 * H floats (needed when any sum is asked
 * for). */
int fl_test_layernorm_bwd_fused(int dtype, const void* dy, const void* x, const float* mean, const float* rstd,
                                const void* g, const void* dres, void* dx, int T, int H, float* dgamma, float* dbeta,
                                float* dsum, float* partial, void* stream);
/* out[n] += sum_t X[t][n] (mode 0); mode 1: out[n] += sum_t X[t][n] *
 * (Y[t][n] - mean[t]) * rstd[t] and out2[n] += sum_t X[t][n].
 * partial: device fp32 scratch of at least ceil(T/256) * N * 2 floats. */
int fl_test_colsum(int dtype, int mode, const void* X, const void* Y, const float* mean, const float* rstd, int T,
                   int N, float* out, float* out2, float* partial, void* stream);
/* Rotary encoding in place on the q and k parts of qkv [T, 3H]; positions
 * from device cu_seqlens [S+1]; table scratch cos/sin: device fp32
 * [max_seqlen * rotary_dim / 2] each; pos scratch: device int32 [T]. */
int fl_test_rope(int dtype, void* qkv, const int32_t* cu_dev, int S, int T, int max_seqlen, int H, int num_heads,
                 int rotary_dim, float base, int32_t* pos, float* cos_t, float* sin_t, void* stream);
/* Attention forward over packed sequences (device cu_seqlens [S+1], device
 * prefix [S] or NULL for causal): qkv [T, 3H] -> o [T, H], lse [T, n_h].
 * pk, pv [num_prefix, H] (bf16, device): P-tuning v2 prefix keys / values in
 * front of every sequence's (num_prefix 0: none). */
int fl_test_attention_fwd(int dtype, const void* qkv, void* o, float* lse, const int32_t* cu_dev,
                          const int32_t* prefix_dev, int T, int S, int max_seqlen, int H, int num_heads,
                          const void* pk, const void* pv, int num_prefix, void* stream);
/* Attention backward: dqkv [T, 3H] from dout [T, H]; delta scratch [T, n_h];
 * rotary_dim 0 disables the inverse rotation, otherwise pos/cos/sin come
 * from fl_test_rope's scratch.  With a prefix, dprefix_part receives the
 * per-sequence prefix gradients, fp32 [2][S][num_prefix][H] (keys, then
 * values).  ds_work (device, ds_bytes >= fl_test_attention_ds_bytes) holds
 * the stored softmax gradient of the bf16 kernels, which dq then reads; NULL:
 * dq recomputes it. */
int fl_test_attention_bwd(int dtype, const void* qkv, const void* o, const float* lse, const void* dout, void* dqkv,
                          float* delta, const int32_t* cu_dev, const int32_t* prefix_dev, const int32_t* pos,
                          const float* cos_t, const float* sin_t, int rotary_dim, int T, int S, int max_seqlen, int H,
                          int num_heads, const void* pk, const void* pv, int num_prefix, float* dprefix_part,
                          void* ds_work, size_t ds_bytes, void* stream);
/* Bytes of ds_work for fl_test_attention_bwd over these host sequence bounds
 * (cu_host [S+1], prefix_host [S] or NULL). */
int fl_test_attention_ds_bytes(const int32_t* cu_host, const int32_t* prefix_host, int S, int num_heads,
                               int num_prefix, size_t* bytes);

#ifdef __cplusplus
}
#endif

#endif /* FLGLM_TESTING_H_ */
