// Single-kernel entry points for per-kernel parity tests (flglm_testing.h).
// Each validates the shape constraints its kernel relies on before any launch.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdarg>
#include <cstdio>

#include "../../include/flglm_testing.h"
#include "kernels.h"

using namespace flglm;

extern "C" const char* fl_last_error(void);
namespace flglm {
int set_error(int code, const char* msg);
}

namespace {
bool al16(const void* p) { return ((uintptr_t)p & 15) == 0; }
int herr(hipError_t e) {
  if (e == hipSuccess) return FL_OK;
  return set_error(FL_ERR_HIP, hipGetErrorString(e));
}
int dtype_ok(int dtype) { return dtype == FL_BF16 || dtype == FL_F32; }
}  // namespace

extern "C" {

int fl_test_gemm(int dtype, int layout, int epi, const void* A, const void* B, void* C, int M, int N, int K,
                 int64_t lda, int64_t ldb, int64_t ldc, const void* bias, const void* R, int64_t ldr, void* C2,
                 int64_t ldc2, const void* Z, int64_t ldz, float* part, int64_t part_bytes, int b_rows,
                 float res_scale, float* colsum, void* stream) {
  if (!dtype_ok(dtype)) return set_error(FL_ERR_ARG, "bad dtype");
  if (!A || !B || !C) return set_error(FL_ERR_NULL, "A / B / C is NULL");
  if (!al16(A) || !al16(B) || !al16(C)) return set_error(FL_ERR_ALIGN, "A / B / C not 16-byte aligned");
  if (M < 0 || N <= 0 || K <= 0) return set_error(FL_ERR_ARG, "bad M / N / K");
  if (N % (dtype == FL_BF16 ? 128 : 64) != 0) return set_error(FL_ERR_ARG, "N not a multiple of the tile width");
  if ((lda | ldb | ldc) % 8 != 0) return set_error(FL_ERR_ARG, "leading dimensions must be multiples of 8");
  bool ok = false;
  switch (layout) {
    case FL_GEMM_NT:
      ok = (epi == FL_EPI_STORE || epi == FL_EPI_BIAS || epi == FL_EPI_BIAS_RES || epi == FL_EPI_BIAS_GELU) &&
           K % 64 == 0 && lda >= K && ldb >= K && ldc >= N;
      break;
    case FL_GEMM_NN:
      ok = (epi == FL_EPI_STORE || epi == FL_EPI_GELU_BWD || epi == FL_EPI_RES) && K % 64 == 0 && lda >= K &&
           ldb >= N && ldc >= N;
      break;
    case FL_GEMM_TN:
      ok = epi == FL_EPI_ACC_F32 && M % 8 == 0 && lda >= M && ldb >= N && ldc >= N;
      break;
    default:
      break;
  }
  if (!ok) return set_error(FL_ERR_ARG, "unsupported layout / epilogue / shape combination");
  if ((epi == FL_EPI_BIAS || epi == FL_EPI_BIAS_RES || epi == FL_EPI_BIAS_GELU) && (!bias || !al16(bias)))
    return set_error(FL_ERR_NULL, "bias missing or misaligned");
  if ((epi == FL_EPI_BIAS_RES || epi == FL_EPI_RES) && (!R || !al16(R) || ldr % 8 || ldr < N))
    return set_error(FL_ERR_NULL, "R missing");
  if (!std::isfinite(res_scale)) return set_error(FL_ERR_ARG, "res_scale not finite");
  if (epi == FL_EPI_BIAS_GELU && (!C2 || !al16(C2) || ldc2 % 8 || ldc2 < N))
    return set_error(FL_ERR_NULL, "C2 missing");
  if (epi == FL_EPI_GELU_BWD && (!Z || !al16(Z) || ldz % 8 || ldz < N)) return set_error(FL_ERR_NULL, "Z missing");
  if (part && (!al16(part) || part_bytes < 0)) return set_error(FL_ERR_ALIGN, "part misaligned");
  if (b_rows < 0) return set_error(FL_ERR_ARG, "b_rows < 0");
  GemmDesc d;
  d.A = A; d.B = B; d.C = C; d.M = M; d.N = N; d.K = K; d.lda = lda; d.ldb = ldb; d.ldc = ldc;
  d.bias = bias; d.R = R; d.ldr = ldr; d.C2 = C2; d.ldc2 = ldc2; d.Z = Z; d.ldz = ldz;
  d.part = part; d.part_bytes = part ? (size_t)part_bytes : 0;
  d.b_rows = b_rows;
  d.res_scale = res_scale;
  if (colsum) {
    if (!al16(colsum)) return set_error(FL_ERR_ALIGN, "colsum misaligned");
    if (!gemm_fuses_colsum((DType)dtype, (GemmLayout)layout, epi, d))
      return set_error(FL_ERR_ARG, "this GEMM does not produce column sums");
    d.colsum = colsum;
  }
  return herr(gemm((DType)dtype, (GemmLayout)layout, epi, d, (hipStream_t)stream));
}

int fl_test_layernorm_fwd(int dtype, const void* x, const void* g, const void* b, void* y, float* mean, float* rstd,
                          int T, int H, float eps, void* stream) {
  if (!dtype_ok(dtype)) return set_error(FL_ERR_ARG, "bad dtype");
  if (!x || !g || !b || !y || !mean || !rstd) return set_error(FL_ERR_NULL, "NULL argument");
  if (T < 0 || H < 256 || H % 256 || H > 4096) return set_error(FL_ERR_ARG, "bad T / H");
  return herr(layernorm_fwd((DType)dtype, x, g, b, y, mean, rstd, T, H, eps, (hipStream_t)stream));
}

int fl_test_layernorm_bwd(int dtype, const void* dy, const void* x, const float* mean, const float* rstd,
                          const void* g, const void* dres, void* dx, int T, int H, void* stream) {
  if (!dtype_ok(dtype)) return set_error(FL_ERR_ARG, "bad dtype");
  if (!dy || !x || !mean || !rstd || !g || !dres || !dx) return set_error(FL_ERR_NULL, "NULL argument");
  if (T < 0 || H < 256 || H % 256 || H > 4096) return set_error(FL_ERR_ARG, "bad T / H");
  return herr(layernorm_bwd_dx((DType)dtype, dy, x, mean, rstd, g, dres, dx, T, H, (hipStream_t)stream));
}

int fl_test_layernorm_bwd_fused(int dtype, const void* dy, const void* x, const float* mean, const float* rstd,
                                const void* g, const void* dres, void* dx, int T, int H, float* dgamma, float* dbeta,
                                float* dsum, float* partial, void* stream) {
  if (!dtype_ok(dtype)) return set_error(FL_ERR_ARG, "bad dtype");
  if (!dy || !x || !mean || !rstd || !g || !dx) return set_error(FL_ERR_NULL, "NULL argument");
  if ((dgamma == nullptr) != (dbeta == nullptr)) return set_error(FL_ERR_ARG, "dgamma and dbeta: both or neither");
  if ((dgamma || dsum) && !partial) return set_error(FL_ERR_NULL, "NULL partial");
  if (T < 0 || H < 256 || H % 256 || H > 4096) return set_error(FL_ERR_ARG, "bad T / H");
  hipStream_t s = (hipStream_t)stream;
  float* pg = dgamma ? partial : nullptr;
  float* pb = dgamma ? partial + (size_t)kLnBlocks * H : nullptr;
  float* po = dsum ? partial + (size_t)2 * kLnBlocks * H : nullptr;
  int rc = herr(layernorm_bwd_fused((DType)dtype, dy, x, mean, rstd, g, dres, dx, T, H, pg, pb, po, s));
  if (!rc && dgamma) rc = herr(colsum_finish(pg, kLnBlocks, H, dgamma, s));
  if (!rc && dgamma) rc = herr(colsum_finish(pb, kLnBlocks, H, dbeta, s));
  if (!rc && dsum) rc = herr(colsum_finish(po, kLnBlocks, H, dsum, s));
  return rc;
}

int fl_test_colsum(int dtype, int mode, const void* X, const void* Y, const float* mean, const float* rstd, int T,
                   int N, float* out, float* out2, float* partial, void* stream) {
  if (!dtype_ok(dtype) || (mode != 0 && mode != 1)) return set_error(FL_ERR_ARG, "bad dtype / mode");
  if (!X || !out || !partial) return set_error(FL_ERR_NULL, "NULL argument");
  if (mode == 1 && (!Y || !mean || !rstd || !out2)) return set_error(FL_ERR_NULL, "NULL argument");
  if (T <= 0 || N <= 0 || N % 8) return set_error(FL_ERR_ARG, "bad T / N");
  hipStream_t s = (hipStream_t)stream;
  const int nb = colsum_blocks(T);
  float* p2 = partial + (size_t)nb * N;
  int rc = herr(colsum_partial((DType)dtype, mode, X, N, Y, mean, rstd, T, N, partial, p2, s));
  if (rc) return rc;
  if ((rc = herr(colsum_finish(partial, nb, N, out, s)))) return rc;
  if (mode == 1) rc = herr(colsum_finish(p2, nb, N, out2, s));
  return rc;
}

int fl_test_rope(int dtype, void* qkv, const int32_t* cu_dev, int S, int T, int max_seqlen, int H, int num_heads,
                 int rotary_dim, float base, int32_t* pos, float* cos_t, float* sin_t, void* stream) {
  if (!dtype_ok(dtype)) return set_error(FL_ERR_ARG, "bad dtype");
  if (!qkv || !cu_dev || !pos || !cos_t || !sin_t) return set_error(FL_ERR_NULL, "NULL argument");
  if (num_heads <= 0 || H % num_heads) return set_error(FL_ERR_ARG, "bad heads");
  const int d = H / num_heads;
  if (rotary_dim < 0 || rotary_dim > d || rotary_dim % 8) return set_error(FL_ERR_ARG, "bad rotary_dim");
  hipStream_t s = (hipStream_t)stream;
  int rc = herr(seq_positions(cu_dev, S, pos, s));
  if (rc) return rc;
  if ((rc = herr(rope_table(cos_t, sin_t, max_seqlen, rotary_dim, base, s)))) return rc;
  return herr(rope_qk((DType)dtype, qkv, 3L * H, pos, cos_t, sin_t, T, H, d, rotary_dim, s));
}

// P-tuning v2 prefix arguments shared by the attention test entries.
int check_prefix(int dtype, const void* pk, const void* pv, int num_prefix) {
  if (num_prefix < 0 || num_prefix > 4096) return set_error(FL_ERR_ARG, "bad num_prefix");
  if (num_prefix && dtype != FL_BF16) return set_error(FL_ERR_ARG, "the prefix needs bf16");
  if (num_prefix && (!pk || !pv || !al16(pk) || !al16(pv))) return set_error(FL_ERR_NULL, "prefix k / v missing");
  return FL_OK;
}

int fl_test_attention_fwd(int dtype, const void* qkv, void* o, float* lse, const int32_t* cu_dev,
                          const int32_t* prefix_dev, int T, int S, int max_seqlen, int H, int num_heads,
                          const void* pk, const void* pv, int num_prefix, void* stream) {
  if (!dtype_ok(dtype)) return set_error(FL_ERR_ARG, "bad dtype");
  if (!qkv || !o || !lse || !cu_dev) return set_error(FL_ERR_NULL, "NULL argument");
  if (num_heads <= 0 || H % num_heads) return set_error(FL_ERR_ARG, "bad heads");
  const int d = H / num_heads;
  if (d != 64 && d != 128) return set_error(FL_ERR_ARG, "head dim must be 64 or 128");
  if (int rc = check_prefix(dtype, pk, pv, num_prefix)) return rc;
  AttnDesc a;
  a.qkv = qkv; a.ld_qkv = 3L * H; a.o = o; a.ld_o = H; a.lse = lse; a.cu_seqlens = cu_dev; a.prefix_len = prefix_dev;
  a.num_seqs = S; a.max_seqlen = max_seqlen; a.num_heads = num_heads; a.head_dim = d; a.hidden = H;
  a.total_tokens = T;
  a.pk = pk; a.pv = pv; a.num_prefix = num_prefix;
  return herr(attn_fwd((DType)dtype, a, (hipStream_t)stream));
}

int fl_test_attention_bwd(int dtype, const void* qkv, const void* o, const float* lse, const void* dout, void* dqkv,
                          float* delta, const int32_t* cu_dev, const int32_t* prefix_dev, const int32_t* pos,
                          const float* cos_t, const float* sin_t, int rotary_dim, int T, int S, int max_seqlen, int H,
                          int num_heads, const void* pk, const void* pv, int num_prefix, float* dprefix_part,
                          void* ds_work, size_t ds_bytes, void* stream) {
  if (!dtype_ok(dtype)) return set_error(FL_ERR_ARG, "bad dtype");
  if (!qkv || !o || !lse || !dout || !dqkv || !delta || !cu_dev) return set_error(FL_ERR_NULL, "NULL argument");
  if (num_heads <= 0 || H % num_heads) return set_error(FL_ERR_ARG, "bad heads");
  const int d = H / num_heads;
  if (d != 64 && d != 128) return set_error(FL_ERR_ARG, "head dim must be 64 or 128");
  if (rotary_dim < 0 || rotary_dim > d || rotary_dim % 32) return set_error(FL_ERR_ARG, "bad rotary_dim");
  if (rotary_dim && (!pos || !cos_t || !sin_t)) return set_error(FL_ERR_NULL, "rotary tables missing");
  if (int rc = check_prefix(dtype, pk, pv, num_prefix)) return rc;
  if (num_prefix && (!dprefix_part || !al16(dprefix_part))) return set_error(FL_ERR_NULL, "dprefix_part missing");
  AttnDesc a;
  a.qkv = qkv; a.ld_qkv = 3L * H; a.o = const_cast<void*>(o); a.ld_o = H; a.lse = const_cast<float*>(lse);
  a.cu_seqlens = cu_dev; a.prefix_len = prefix_dev; a.num_seqs = S; a.max_seqlen = max_seqlen;
  a.num_heads = num_heads; a.head_dim = d; a.hidden = H; a.total_tokens = T;
  a.dout = dout; a.ld_dout = H; a.delta = delta; a.dqkv = dqkv; a.ld_dqkv = 3L * H;
  a.pos = pos; a.cos_t = cos_t; a.sin_t = sin_t; a.rotary_dim = rotary_dim;
  a.pk = pk; a.pv = pv; a.num_prefix = num_prefix; a.dprefix_part = dprefix_part;
  if (ds_work) {
    // [S + 1] int64 offsets (256-byte aligned), then the tiles; the tile
    // count needs the host bounds, so only the size is checked here
    if (dtype != FL_BF16) return set_error(FL_ERR_ARG, "stored dS needs bf16");
    const size_t head = attn_ds_off_bytes(S);
    if (ds_bytes < head || ((uintptr_t)ds_work & 255)) return set_error(FL_ERR_WORKSPACE, "ds_work too small or unaligned");
    a.ds_off = static_cast<int64_t*>(ds_work);
    a.ds = static_cast<char*>(ds_work) + head;
    // the tile count from the device bounds, checked before anything writes
    // tiles
    hipStream_t sm = (hipStream_t)stream;
    int64_t total = 0;
    if (hipError_t e = attn_ds_offsets(a, sm); e != hipSuccess) return herr(e);
    if (hipError_t e = hipMemcpyAsync(&total, a.ds_off + S, sizeof(total), hipMemcpyDeviceToHost, sm); e != hipSuccess)
      return herr(e);
    if (hipError_t e = hipStreamSynchronize(sm); e != hipSuccess) return herr(e);
    if (total < 0 || ds_bytes < head + (size_t)total * kAttnDsTileBytes)
      return set_error(FL_ERR_WORKSPACE, "ds_work smaller than the stored dS needs");
  }
  return herr(attn_bwd((DType)dtype, a, (hipStream_t)stream));
}

int fl_test_attention_ds_bytes(const int32_t* cu_host, const int32_t* prefix_host, int S, int num_heads,
                               int num_prefix, size_t* bytes) {
  if (!cu_host || !bytes) return set_error(FL_ERR_NULL, "NULL argument");
  if (S < 1 || num_heads < 1 || num_prefix < 0) return set_error(FL_ERR_ARG, "bad sizes");
  *bytes = attn_ds_off_bytes(S) + attn_ds_tiles(cu_host, prefix_host, S, num_heads, num_prefix) * kAttnDsTileBytes;
  return FL_OK;
}

}  // extern "C"
