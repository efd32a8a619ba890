// Host-side launch functions of the device kernels (internal to the library).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace flglm {

enum DType : int { DT_BF16 = 0, DT_F32 = 1 };
enum GemmLayout : int { GEMM_NT = 0, GEMM_NN = 1, GEMM_TN = 2 };

// C[m, n] (op)= sum_k A(m, k) B(n, k); see gemm.hip for layouts and epilogues.
struct GemmDesc {
  const void* A = nullptr;
  const void* B = nullptr;
  void* C = nullptr;
  int M = 0, N = 0, K = 0;
  long lda = 0, ldb = 0, ldc = 0;
  const void* bias = nullptr;
  const void* R = nullptr;
  long ldr = 0;
  void* C2 = nullptr;
  long ldc2 = 0;
  const void* Z = nullptr;
  long ldz = 0;
  // Optional fp32 scratch for splitting the reduction of a partial last
  // round of tiles (bf16 LDS-DMA kernel); null = never split.
  float* part = nullptr;
  size_t part_bytes = 0;
  // Rows B really has (the N index for NT, the reduction index for NN / TN);
  // rows at or past it read as zero.  0 = as many as the shape implies.
  int b_rows = 0;
  // Scale of R in EPI_BIAS_RES and EPI_RES (1: plain residual add).
  float res_scale = 1.f;
  // EPI_GELU_BWD where gemm_fuses_colsum() holds: fp32 [ceil(M / 256)][N]
  // receives, per 256-row block, the column sums of the stored C (the
  // layout colsum_partial writes, so colsum_finish completes them).
  float* colsum = nullptr;
};
// Rows of B a kernel may read for a layout and shape.
inline int gemm_b_rows(bool b_kcontig, const GemmDesc& d) {
  const int full = b_kcontig ? d.N : d.K;
  return d.b_rows > 0 && d.b_rows < full ? d.b_rows : full;
}
// Scratch that lets gemm() split the partial last round of tiles (one
// 256 KB slice per compute unit).
size_t gemm_part_bytes();
enum GemmEpi : int {
  EPI_STORE = 0,      // C = acc
  EPI_BIAS = 1,       // C = acc + bias
  EPI_BIAS_RES = 2,   // C = acc + bias + R
  EPI_BIAS_GELU = 3,  // C = z = acc + bias (skipped when C is null); C2 = gelu(z)
  EPI_GELU_BWD = 4,   // C = acc * gelu'(Z)
  EPI_ACC_F32 = 5,    // Cf += acc (fp32 output)
  EPI_RES = 6,        // C = acc + res_scale * R
};
hipError_t gemm(DType dt, GemmLayout layout, int epi, const GemmDesc& d, hipStream_t st);
// bf16 LDS-DMA kernel (gemm_bf16.hip), used by gemm() for the shapes it takes.
bool gemm_bf16_dma_ok(GemmLayout layout, const GemmDesc& d);
// Whether gemm() fills d.colsum for this call (bf16 GeLU' input-gradient
// GEMMs on the LDS-DMA kernel); otherwise the caller sums the columns itself.
bool gemm_fuses_colsum(DType dt, GemmLayout layout, int epi, const GemmDesc& d);
hipError_t gemm_bf16_dma(GemmLayout layout, int epi, const GemmDesc& d, hipStream_t st);

// Batch bookkeeping: position of every packed row inside its own sequence.
hipError_t seq_positions(const int32_t* cu_seqlens, int num_seqs, int32_t* pos, hipStream_t st);
// GLM 2-D positions (context length ctx[s], or the whole sequence when ctx is null).
hipError_t seq_positions_2d(const int32_t* cu_seqlens, const int32_t* ctx, int num_seqs, int32_t* p1, int32_t* p2,
                            hipStream_t st);
// cos / sin (p * theta_i), theta_i = base^(-2i/r), p < max_pos, i < r/2 (computed in double).
hipError_t rope_table(float* cos_t, float* sin_t, int max_pos, int rotary_dim, float base, hipStream_t st);
// In-place rotation of the q and k parts of qkv [T, 3H] (row stride ld):
// dims [0, rotary_dim) of every head by pos; with pos2 (GLM 2-D positions)
// also dims [rotary_dim, 2 rotary_dim) by pos2.  sign -1 rotates back.
hipError_t rope_qk(DType dt, void* qkv, long ld, const int32_t* pos, const float* cos_t, const float* sin_t,
                   int T, int H, int head_dim, int rotary_dim, hipStream_t st, float sign = 1.f,
                   const int32_t* pos2 = nullptr);

// LayerNorm forward: y = (x - mean) * rstd * g + b, saving mean and rstd.
hipError_t layernorm_fwd(DType dt, const void* x, const void* g, const void* b, void* y, float* mean,
                         float* rstd, int T, int H, float eps, hipStream_t st);
// LayerNorm backward (input grad only): dx = dres + rstd*(dxh - mean(dxh) - xh*mean(dxh*xh)),
// dxh = dy * g, xh = (x - mean) * rstd.  dres may alias nothing written here.
hipError_t layernorm_bwd_dx(DType dt, const void* dy, const void* x, const float* mean, const float* rstd,
                            const void* g, const void* dres, void* dx, int T, int H, hipStream_t st);

// LayerNorm backward fused with its column sums: dx as layernorm_bwd_dx, and
// per block of rows (kLnBlocks blocks of T / kLnBlocks rows; partials
// [kLnBlocks][H] fp32, completed by colsum_finish): pg, pb = the gain / shift
// gradient sums (sum dy * xh, sum dy; both or neither), pout = the sum of
// the stored dx (or null).  H <= 4096.
constexpr int kLnBlocks = 512;
hipError_t layernorm_bwd_fused(DType dt, const void* dy, const void* x, const float* mean, const float* rstd,
                               const void* g, const void* dres, void* dx, int T, int H, float* pg, float* pb,
                               float* pout, hipStream_t st);

// Deterministic column sums over T rows, two stages.  Stage 1 writes
// partial[blk][n] for row blocks of kColsumRows rows; stage 2 adds the sum
// over blocks (fixed order) into out[n] (fp32, +=).
constexpr int kColsumRows = 256;
inline int colsum_blocks(int T) { return (T + kColsumRows - 1) / kColsumRows; }
// mode 0: sum_t X[t][n].  mode 1: sum_t X[t][n] * (Y[t][n] - mean[t]) * rstd[t]
// (the LayerNorm gain gradient), written to partial; mode 1 also writes the
// plain sum of X to partial2.
hipError_t colsum_partial(DType dt, int mode, const void* X, long ldx, const void* Y, const float* mean,
                          const float* rstd, int T, int N, float* partial, float* partial2, hipStream_t st);
hipError_t colsum_finish(const float* partial, int nblk, int N, float* out, hipStream_t st);
// colsum_finish of up to three partial arrays of one shape in one launch.
hipError_t colsum_finish_n(const float* const* partials, float* const* outs, int count, int nblk, int N,
                           hipStream_t st);

// P-tuning v2 prefix gradients: out_k += sum_s part[0][s], out_v += sum_s
// part[1][s] over n = num_prefix * hidden elements (n % 4 == 0; fixed order).
hipError_t prefix_grad_reduce(const float* part, int S, long n, float* out_k, float* out_v, hipStream_t st);

// Attention over packed ragged sequences.  qkv rows are [q | k | v] (each H
// wide, head h at columns h*d); o is [T, H]; lse is [T, nh] fp32.
struct AttnDesc {
  const void* qkv = nullptr;
  long ld_qkv = 0;
  void* o = nullptr;
  long ld_o = 0;
  float* lse = nullptr;  // natural-log sum-exp of scaled scores, [T, nh]
  const int32_t* cu_seqlens = nullptr;  // device [S+1]
  const int32_t* prefix_len = nullptr;  // device [S] or null (causal)
  int num_seqs = 0, max_seqlen = 0, num_heads = 0, head_dim = 0, hidden = 0;
  // backward
  const void* dout = nullptr;
  long ld_dout = 0;
  float* delta = nullptr;  // [T, nh] scratch: rowsum(dO * O)
  void* dqkv = nullptr;    // [T, 3H]
  long ld_dqkv = 0;
  // Inverse rotary of dq, dk fused into the kernels' epilogues, over dims
  // [0, rotary_dim) with the row's index inside its sequence as the
  // position (0 = no rotation).
  const int32_t* pos = nullptr;
  const float* cos_t = nullptr;
  const float* sin_t = nullptr;
  int rotary_dim = 0;
  int total_tokens = 0;
  // P-tuning v2 prefix (bf16 kernels): num_prefix rows of keys pk and values
  // pv ([num_prefix, hidden], head h at columns h*d, not rotated) in front of
  // every sequence's keys, visible to all of its queries.  The backward
  // writes per-sequence prefix gradients to dprefix_part, fp32
  // [2][num_seqs][num_prefix][hidden] (keys, then values).
  const void* pk = nullptr;
  const void* pv = nullptr;
  int num_prefix = 0;
  float* dprefix_part = nullptr;
  // Backward (bf16 kernels): storage for the softmax gradient dS, 64 x 64
  // bf16 tiles (attn_ds_tiles of them), and ds_off, device int64 [S + 1]
  // scratch for their per-sequence offsets.  Null ds: the dq kernel
  // recomputes S and dP instead of reading dS.
  void* ds = nullptr;
  int64_t* ds_off = nullptr;
  // With ds: per 64-row tile of each sequence, the column sums of the stored
  // dq | dk | dv rows (fp32 [tile rows][3 hidden]; tile rows numbered
  // sequence after sequence, tile_base (device int32 [S + 1] scratch)
  // receives each sequence's first); null: not formed.
  float* bias_part = nullptr;
  int32_t* tile_base = nullptr;
};
// Tiles of stored dS a backward over these (host) sequence bounds needs:
// per sequence and head, one per (64-query tile, 64-key tile) pair holding a
// visible pair, prefix key tiles included.
size_t attn_ds_tiles(const int32_t* cu_host, const int32_t* prefix_host, int num_seqs, int num_heads,
                     int num_prefix);
constexpr size_t kAttnDsTileBytes = 64 * 64 * 2;
// Fills a.ds_off from the device sequence bounds (ds_off[S] = the total).
hipError_t attn_ds_offsets(const AttnDesc& a, hipStream_t st);
// Bytes of the ds_off table (S + 1 int64), rounded up to 256.
inline size_t attn_ds_off_bytes(int num_seqs) { return ((size_t)(num_seqs + 1) * 8 + 255) / 256 * 256; }
hipError_t attn_fwd(DType dt, const AttnDesc& a, hipStream_t st);
hipError_t attn_bwd(DType dt, const AttnDesc& a, hipStream_t st);
// delta[t][h] = rowsum(dO * O), the backward pre-pass.
hipError_t attn_delta(DType dt, const AttnDesc& a, hipStream_t st);
// bf16 LDS-DMA kernels (attention_bf16.hip), used by attn_fwd / attn_bwd.
bool attn_bf16_ok(const AttnDesc& a);
hipError_t attn_fwd_bf16(const AttnDesc& a, hipStream_t st);
hipError_t attn_bwd_bf16(const AttnDesc& a, hipStream_t st);

// Client packing: client tensor [Lmax, nseq, H] (sequence-first) <-> packed
// rows of sequences s0 .. s0+nseq-1.  Unpacking zero-fills padded positions.
hipError_t pack_client(DType dt, const void* client, void* packed, const int32_t* cu_dev, int s0, int nseq,
                       int Lmax, int H, bool unpack, hipStream_t st);

}  // namespace flglm
