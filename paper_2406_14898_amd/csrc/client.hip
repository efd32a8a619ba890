// The client side of the split model around the server stack (Section 3.1,
// Model Split): the embedding layer in front of block 0 and the final linear
// layer with the cross-entropy loss behind block N-1, forward and backward.
// The client's two blocks are one-block stacks of the same engine.
//
// Token ids and labels are host data (the client's own tokens); they travel
// to the device through a pinned staging ring, like the server's batch plan.
// The embedding gradient is a deterministic segmented sum: the host orders
// the tokens by id (counting sort, ties in token order) and the device adds
// each id's rows in that order, with no atomics.
//
// An optional final LayerNorm (ChatGLM-6B's, not in the paper's formula) can
// sit in front of the linear layer; its output, statistics and the gradient
// arriving at it live in the workspace.
//
// The vocabulary is padded to a multiple of the 256-wide GEMM tile inside
// the workspace: the logits buffer is [T, V_pad]; rows of the weight past V
// are never read (the GEMM reads them as zero), and the padded columns take
// no part in the softmax and get a zero gradient.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <new>
#include <vector>

#include "../../include/flglm.h"
#include "common.h"
#include "kernels.h"

namespace flglm {
int set_error(int code, const char* msg);
}

using namespace flglm;

struct fl_client {
  fl_client_desc d;
  int E = 2;       // element bytes
  long vpad = 0;   // vocabulary padded to the GEMM tile
  static constexpr int kRing = 4;
  void* stage[kRing] = {};
  size_t stage_cap[kRing] = {};
  hipEvent_t ev[kRing] = {};
  bool ev_made[kRing] = {};
  bool ev_used[kRing] = {};
  int next = 0;
};

namespace {

constexpr int kThreads = 256;
constexpr long kVocabTile = 256;
constexpr int kLossThreads = 256;

long align256(long x) { return (x + 255) & ~255L; }
bool al16(const void* p) { return ((uintptr_t)p & 15) == 0; }
bool overlap(const void* a, size_t na, const void* b, size_t nb) {
  const uintptr_t x = (uintptr_t)a, y = (uintptr_t)b;
  return x < y + nb && y < x + na;
}
int herr(hipError_t e) { return e == hipSuccess ? FL_OK : set_error(FL_ERR_HIP, hipGetErrorString(e)); }
#define CK(expr)                                \
  do {                                          \
    int rc_ = herr(expr);                       \
    if (rc_ != FL_OK) return rc_;               \
  } while (0)

// Workspace carving for T tokens.
struct ClientWs {
  char* logits;   // [T, V_pad] elements (bf16 or fp32)
  float* lse;     // [T]
  int32_t* labels;  // [T]
  int32_t* ids;     // [T]
  int32_t* plan;    // order [T] | segment starts [T + 1] | segment ids [T]
  char* hn;         // final LayerNorm output [T, H]
  char* dhn;        // gradient at the final LayerNorm output [T, H]
  float* mean;      // final LayerNorm statistics [T]
  float* rstd;
  float* ln_part;   // column-sum partials of the LayerNorm gain / shift gradients
  float* ln_part2;
  float* part;      // GEMM split-reduction scratch
  size_t part_bytes;
  size_t total;
};

ClientWs carve(const fl_client* c, long T, char* base) {
  ClientWs w;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    char* p = base ? base + off : nullptr;
    off = align256(off + bytes);
    return p;
  };
  w.logits = take((size_t)T * c->vpad * c->E);
  w.lse = (float*)take((size_t)T * 4);
  w.labels = (int32_t*)take((size_t)T * 4);
  w.ids = (int32_t*)take((size_t)T * 4);
  w.plan = (int32_t*)take((size_t)(3 * T + 1) * 4);
  const size_t th = (size_t)T * c->d.hidden * c->E;
  w.hn = take(th);
  w.dhn = take(th);
  w.mean = (float*)take((size_t)T * 4);
  w.rstd = (float*)take((size_t)T * 4);
  const size_t cp = (size_t)colsum_blocks((int)T) * c->d.hidden * 4;
  w.ln_part = (float*)take(cp);
  w.ln_part2 = (float*)take(cp);
  w.part_bytes = gemm_part_bytes();
  w.part = (float*)take(w.part_bytes);
  w.total = off;
  return w;
}

// Pinned staging: copies `bytes` of host data to `dst` on `stream`.  A slot
// is reused only after its previous copy has completed.
int upload(fl_client* c, const void* src, size_t bytes, void* dst, hipStream_t stream) {
  const int k = c->next;
  c->next = (c->next + 1) % fl_client::kRing;
  if (!c->ev_made[k]) {
    CK(hipEventCreateWithFlags(&c->ev[k], hipEventDisableTiming));
    c->ev_made[k] = true;
  }
  if (c->ev_used[k]) CK(hipEventSynchronize(c->ev[k]));
  if (c->stage_cap[k] < bytes) {
    if (c->stage[k]) CK(hipHostFree(c->stage[k]));
    c->stage[k] = nullptr;
    c->stage_cap[k] = 0;
    const size_t cap = std::max(bytes, (size_t)4096);
    CK(hipHostMalloc(&c->stage[k], cap, hipHostMallocDefault));
    c->stage_cap[k] = cap;
  }
  std::memcpy(c->stage[k], src, bytes);
  CK(hipMemcpyAsync(dst, c->stage[k], bytes, hipMemcpyHostToDevice, stream));
  CK(hipEventRecord(c->ev[k], stream));
  c->ev_used[k] = true;
  return FL_OK;
}

// ---------------------------------------------------------------------------
// Kernels
// ---------------------------------------------------------------------------

// out[t] = table[ids[t]]: one workgroup per token, 16-byte copies.
__global__ void __launch_bounds__(kThreads) embed_gather_kernel(const char* table, const int32_t* ids, long row_bytes,
                                                                char* out) {
  const long t = blockIdx.x;
  const u32x4* src = reinterpret_cast<const u32x4*>(table + (long)ids[t] * row_bytes);
  u32x4* dst = reinterpret_cast<u32x4*>(out + t * row_bytes);
  for (long i = threadIdx.x; i < row_bytes / 16; i += kThreads) dst[i] = src[i];
}

// dtable[id] += sum of dout over the tokens of id's segment, in token order:
// one workgroup per (segment, 1024 columns), four columns per lane.
template <typename T>
__global__ void __launch_bounds__(kThreads) embed_grad_kernel(const int32_t* order, const int32_t* seg_start,
                                                              const int32_t* seg_id, const T* dout, int H,
                                                              float* dtable) {
  const int s = blockIdx.x;
  const int c = (blockIdx.y * kThreads + threadIdx.x) * 4;
  if (c >= H) return;
  float acc[4] = {0.f, 0.f, 0.f, 0.f};
  for (int i = seg_start[s]; i < seg_start[s + 1]; ++i) {
    Vec4<T> v;
    v.load(dout + (long)order[i] * H + c);
#pragma unroll
    for (int k = 0; k < 4; ++k) acc[k] += v.get(k);
  }
  float* dst = dtable + (long)seg_id[s] * H + c;
  Vec4<float> o;
  o.load(dst);
  float r[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) r[k] = o.get(k) + acc[k];
  o.set(r);
  o.store(dst);
}

// (max, sum of exp(x - max)) pairs: combining keeps the larger maximum.
__device__ __forceinline__ void lse_merge(float& m, float& s, float m2, float s2) {
  if (m2 == -INFINITY) return;
  if (m == -INFINITY) {
    m = m2;
    s = s2;
    return;
  }
  const float mx = fmaxf(m, m2);
  s = s * __expf(m - mx) + s2 * __expf(m2 - mx);
  m = mx;
}

// Row t of the logits: log-sum-exp over the V real columns and the token's
// loss lse - logit[label] (0 for an unlabelled token).  Eight columns per
// lane per pass, one running (max, sum) per lane, then a workgroup merge.
template <typename T>
__global__ void __launch_bounds__(kThreads) ce_fwd_kernel(const T* logits, long ld, int V, const int32_t* labels,
                                                          float* lse, float* loss_tok) {
  const long t = blockIdx.x;
  const T* row = logits + t * ld;
  float m = -INFINITY, s = 0.f;
  for (int j0 = threadIdx.x * 8; j0 < V; j0 += kThreads * 8) {
    Vec8<T> v;
    v.load(row + j0);
    float x[8];
    float mx = -INFINITY;
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      x[k] = j0 + k < V ? v.get(k) : -INFINITY;
      mx = fmaxf(mx, x[k]);
    }
    float sum = 0.f;
#pragma unroll
    for (int k = 0; k < 8; ++k) sum += __expf(x[k] - mx);
    lse_merge(m, s, mx, sum);
  }
  // wave merge, then across the four waves through LDS
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) {
    const float m2 = __shfl_xor(m, off), s2 = __shfl_xor(s, off);
    lse_merge(m, s, m2, s2);
  }
  __shared__ float sm[kThreads / 64], ss[kThreads / 64];
  const int wave = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) {
    sm[wave] = m;
    ss[wave] = s;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    float M = sm[0], S = ss[0];
    for (int w = 1; w < kThreads / 64; ++w) lse_merge(M, S, sm[w], ss[w]);
    const float l = M + logf(S);
    lse[t] = l;
    const int lab = labels[t];
    loss_tok[t] = lab >= 0 ? l - to_f32(row[lab]) : 0.f;
  }
}

// In place: logits -> grad_scale * (softmax - onehot(label)) on the real
// columns of labelled rows, 0 elsewhere.
template <typename T>
__global__ void __launch_bounds__(kThreads) ce_bwd_kernel(T* logits, long ld, int V, const int32_t* labels,
                                                          const float* lse, float scale) {
  const long t = blockIdx.x;
  T* row = logits + t * ld;
  const int lab = labels[t];
  const float l = lse[t];
  for (long j0 = threadIdx.x * 8; j0 < ld; j0 += kThreads * 8) {
    Vec8<T> v;
    v.load(row + j0);
    float g[8];
#pragma unroll
    for (int k = 0; k < 8; ++k) {
      const long j = j0 + k;
      g[k] = (lab >= 0 && j < V) ? (__expf(v.get(k) - l) - (j == lab ? 1.f : 0.f)) * scale : 0.f;
    }
    v.set(g);
    v.store(row + j0);
  }
}

// loss_sum = sum of loss_tok: each lane adds a fixed stride of tokens, then
// a fixed-order tree (deterministic).
__global__ void __launch_bounds__(kLossThreads) loss_sum_kernel(const float* loss_tok, long T, float* out) {
  __shared__ float red[kLossThreads];
  float a = 0.f;
  for (long i = threadIdx.x; i < T; i += kLossThreads) a += loss_tok[i];
  red[threadIdx.x] = a;
  __syncthreads();
  for (int w = kLossThreads / 2; w >= 1; w >>= 1) {
    if (threadIdx.x < w) red[threadIdx.x] += red[threadIdx.x + w];
    __syncthreads();
  }
  if (threadIdx.x == 0) *out = red[0];
}

DType dt_of(const fl_client* c) { return c->d.dtype == FL_BF16 ? DT_BF16 : DT_F32; }

int check_common(const fl_client* c, long T, void* ws, size_t ws_bytes) {
  if (!c) return set_error(FL_ERR_NULL, "client handle is NULL");
  if (T < 1 || T > (1L << 26)) return set_error(FL_ERR_ARG, "token count must be in [1, 2^26]");
  if (!ws) return set_error(FL_ERR_NULL, "workspace is NULL");
  if (!al16(ws)) return set_error(FL_ERR_ALIGN, "workspace is not 16-byte aligned");
  if (ws_bytes < carve(c, T, nullptr).total) return set_error(FL_ERR_WORKSPACE, "workspace too small");
  return FL_OK;
}

}  // namespace

extern "C" {

int fl_client_create(const fl_client_desc* desc, fl_client** out) {
  if (!desc || !out) return set_error(FL_ERR_NULL, "desc / out is NULL");
  *out = nullptr;
  if (desc->dtype != FL_BF16 && desc->dtype != FL_F32) return set_error(FL_ERR_SHAPE, "dtype must be bf16 or fp32");
  if (desc->vocab < 8 || desc->vocab % 8 || desc->vocab > (1 << 24))
    return set_error(FL_ERR_SHAPE, "vocab must be a multiple of 8 in [8, 2^24]");
  if (desc->hidden < 256 || desc->hidden % 256 || desc->hidden > 16384)
    return set_error(FL_ERR_SHAPE, "hidden must be a multiple of 256 in [256, 16384]");
  if (!(desc->ln_eps >= 0.f) || !std::isfinite(desc->ln_eps)) return set_error(FL_ERR_SHAPE, "ln_eps must be >= 0");
  // no exception may leave a C entry point: a failed allocation is an error code
  fl_client* c = new (std::nothrow) fl_client;
  if (!c) return set_error(FL_ERR_NOMEM, "out of host memory for the client handle");
  c->d = *desc;
  c->E = desc->dtype == FL_BF16 ? 2 : 4;
  c->vpad = (desc->vocab + kVocabTile - 1) / kVocabTile * kVocabTile;
  *out = c;
  return FL_OK;
}

int fl_client_destroy(fl_client* c) {
  if (!c) return FL_OK;
  for (int k = 0; k < fl_client::kRing; ++k) {
    if (c->ev_used[k]) (void)hipEventSynchronize(c->ev[k]);
    if (c->ev_made[k]) (void)hipEventDestroy(c->ev[k]);
    if (c->stage[k]) (void)hipHostFree(c->stage[k]);
  }
  delete c;
  return FL_OK;
}

int fl_client_workspace_bytes(const fl_client* c, int64_t T, size_t* bytes) {
  if (!c || !bytes) return set_error(FL_ERR_NULL, "NULL argument");
  if (T < 1 || T > (1L << 26)) return set_error(FL_ERR_ARG, "token count must be in [1, 2^26]");
  *bytes = carve(c, T, nullptr).total;
  return FL_OK;
}

int fl_embedding_forward(fl_client* c, const void* table, const int32_t* ids, int64_t T, void* out, void* workspace,
                         size_t workspace_bytes, void* stream) {
  if (int rc = check_common(c, T, workspace, workspace_bytes)) return rc;
  if (!table || !ids || !out) return set_error(FL_ERR_NULL, "table / ids / out is NULL");
  if (!al16(table) || !al16(out)) return set_error(FL_ERR_ALIGN, "table / out not 16-byte aligned");
  const size_t row = (size_t)c->d.hidden * c->E;
  if (overlap(out, T * row, table, c->d.vocab * row)) return set_error(FL_ERR_ALIAS, "out overlaps the table");
  if (overlap(out, T * row, workspace, workspace_bytes)) return set_error(FL_ERR_ALIAS, "out overlaps the workspace");
  for (long t = 0; t < T; ++t)
    if (ids[t] < 0 || ids[t] >= c->d.vocab) return set_error(FL_ERR_ARG, "a token id is outside [0, vocab)");
  const ClientWs w = carve(c, T, (char*)workspace);
  hipStream_t s = (hipStream_t)stream;
  if (int rc = upload(c, ids, (size_t)T * 4, w.ids, s)) return rc;
  hipLaunchKernelGGL(embed_gather_kernel, dim3((unsigned)T), dim3(kThreads), 0, s, (const char*)table, w.ids,
                     (long)row, (char*)out);
  return herr(hipGetLastError());
}

int fl_embedding_backward(fl_client* c, const int32_t* ids, int64_t T, const void* dout, float* dtable,
                          void* workspace, size_t workspace_bytes, void* stream) {
  if (int rc = check_common(c, T, workspace, workspace_bytes)) return rc;
  if (!ids || !dout || !dtable) return set_error(FL_ERR_NULL, "ids / dout / dtable is NULL");
  if (!al16(dout) || !al16(dtable)) return set_error(FL_ERR_ALIGN, "dout / dtable not 16-byte aligned");
  const long V = c->d.vocab, H = c->d.hidden;
  if (overlap(dtable, V * H * 4, dout, T * H * c->E) || overlap(dtable, V * H * 4, workspace, workspace_bytes))
    return set_error(FL_ERR_ALIAS, "dtable overlaps dout / the workspace");
  // counting sort of the tokens by id, ties in token order
  std::vector<int32_t> count(V + 1, 0);
  for (long t = 0; t < T; ++t) {
    if (ids[t] < 0 || ids[t] >= V) return set_error(FL_ERR_ARG, "a token id is outside [0, vocab)");
    ++count[ids[t] + 1];
  }
  for (long v = 0; v < V; ++v) count[v + 1] += count[v];
  std::vector<int32_t> plan(3 * T + 1);
  int32_t* order = plan.data();
  int32_t* seg = order + T;
  std::vector<int32_t> fill(count.begin(), count.end() - 1);
  for (long t = 0; t < T; ++t) order[fill[ids[t]]++] = (int32_t)t;
  int nseg = 0;
  for (long v = 0; v < V; ++v)
    if (count[v + 1] > count[v]) {
      seg[nseg] = count[v];
      ++nseg;
    }
  seg[nseg] = (int32_t)T;
  int32_t* seg_id = seg + nseg + 1;
  for (long v = 0, k = 0; v < V; ++v)
    if (count[v + 1] > count[v]) seg_id[k++] = (int32_t)v;
  const ClientWs w = carve(c, T, (char*)workspace);
  hipStream_t s = (hipStream_t)stream;
  const size_t plan_ints = (size_t)T + nseg + 1 + nseg;
  if (int rc = upload(c, plan.data(), plan_ints * 4, w.plan, s)) return rc;
  const int32_t* d_order = w.plan;
  const int32_t* d_seg = w.plan + T;
  const int32_t* d_segid = d_seg + nseg + 1;
  const dim3 grid((unsigned)nseg, (unsigned)((H / 4 + kThreads - 1) / kThreads));
  if (c->d.dtype == FL_BF16)
    hipLaunchKernelGGL(embed_grad_kernel<bf16>, grid, dim3(kThreads), 0, s, d_order, d_seg, d_segid,
                       (const bf16*)dout, (int)H, dtable);
  else
    hipLaunchKernelGGL(embed_grad_kernel<float>, grid, dim3(kThreads), 0, s, d_order, d_seg, d_segid,
                       (const float*)dout, (int)H, dtable);
  return herr(hipGetLastError());
}

// The final LayerNorm's arguments: both or neither, hidden <= 4096, eps > 0.
int check_final_ln(const fl_client* c, const void* g, const void* b) {
  if (!g && !b) return FL_OK;
  if (!g || !b) return set_error(FL_ERR_NULL, "final LayerNorm gain / shift: both or neither");
  if (!al16(g) || !al16(b)) return set_error(FL_ERR_ALIGN, "final LayerNorm parameters not 16-byte aligned");
  if (c->d.hidden > 4096) return set_error(FL_ERR_SHAPE, "the final LayerNorm supports hidden <= 4096");
  if (!(c->d.ln_eps > 0.f)) return set_error(FL_ERR_SHAPE, "the final LayerNorm needs ln_eps > 0");
  return FL_OK;
}

int fl_lm_head_forward(fl_client* c, const void* h, const void* ln_g, const void* ln_b, const void* w_vocab,
                       const int32_t* labels, int64_t T, float* loss_tok, float* loss_sum, void* workspace,
                       size_t workspace_bytes, void* stream) {
  if (int rc = check_common(c, T, workspace, workspace_bytes)) return rc;
  if (!h || !w_vocab || !labels || !loss_tok || !loss_sum) return set_error(FL_ERR_NULL, "NULL argument");
  if (int rc = check_final_ln(c, ln_g, ln_b)) return rc;
  if (!al16(h) || !al16(w_vocab) || !al16(loss_tok) || ((uintptr_t)loss_sum & 3))
    return set_error(FL_ERR_ALIGN, "h / w / loss_tok not 16-byte aligned");
  if (overlap(loss_tok, T * 4, workspace, workspace_bytes) || overlap(loss_sum, 4, workspace, workspace_bytes) ||
      overlap(loss_tok, T * 4, loss_sum, 4))
    return set_error(FL_ERR_ALIAS, "loss outputs overlap each other or the workspace");
  for (long t = 0; t < T; ++t)
    if (labels[t] >= c->d.vocab) return set_error(FL_ERR_ARG, "a label is >= vocab");
  const ClientWs w = carve(c, T, (char*)workspace);
  hipStream_t s = (hipStream_t)stream;
  if (int rc = upload(c, labels, (size_t)T * 4, w.labels, s)) return rc;
  const int H = c->d.hidden;
  const void* hin = h;
  if (ln_g) {
    CK(layernorm_fwd(dt_of(c), h, ln_g, ln_b, w.hn, w.mean, w.rstd, (int)T, H, c->d.ln_eps, s));
    hin = w.hn;
  }
  GemmDesc g;
  g.A = hin; g.B = w_vocab; g.C = w.logits;
  g.M = (int)T; g.N = (int)c->vpad; g.K = H;
  g.lda = H; g.ldb = H; g.ldc = c->vpad;
  g.b_rows = (int)c->d.vocab;
  g.part = w.part; g.part_bytes = w.part_bytes;
  CK(gemm(dt_of(c), GEMM_NT, EPI_STORE, g, s));
  if (c->d.dtype == FL_BF16)
    hipLaunchKernelGGL(ce_fwd_kernel<bf16>, dim3((unsigned)T), dim3(kThreads), 0, s, (const bf16*)w.logits,
                       c->vpad, (int)c->d.vocab, w.labels, w.lse, loss_tok);
  else
    hipLaunchKernelGGL(ce_fwd_kernel<float>, dim3((unsigned)T), dim3(kThreads), 0, s, (const float*)w.logits,
                       c->vpad, (int)c->d.vocab, w.labels, w.lse, loss_tok);
  CK(hipGetLastError());
  hipLaunchKernelGGL(loss_sum_kernel, dim3(1), dim3(kLossThreads), 0, s, loss_tok, (long)T, loss_sum);
  return herr(hipGetLastError());
}

int fl_lm_head_backward(fl_client* c, const void* h, const void* ln_g, const void* w_vocab, int64_t T,
                        float grad_scale, void* dh, float* dln_g, float* dln_b, float* dw_vocab, void* workspace,
                        size_t workspace_bytes, void* stream) {
  if (int rc = check_common(c, T, workspace, workspace_bytes)) return rc;
  if (!h || !w_vocab || !dh) return set_error(FL_ERR_NULL, "h / w / dh is NULL");
  if (ln_g && (!al16(ln_g) || c->d.hidden > 4096 || !(c->d.ln_eps > 0.f)))
    return set_error(FL_ERR_ARG, "final LayerNorm gain misaligned, or hidden / ln_eps unsupported");
  if (!ln_g && (dln_g || dln_b)) return set_error(FL_ERR_ARG, "LayerNorm gradients without a final LayerNorm");
  if ((dln_g == nullptr) != (dln_b == nullptr)) return set_error(FL_ERR_NULL, "dln_g / dln_b: both or neither");
  if ((dln_g && !al16(dln_g)) || (dln_b && !al16(dln_b))) return set_error(FL_ERR_ALIGN, "dln not aligned");
  if (!al16(h) || !al16(w_vocab) || !al16(dh) || (dw_vocab && !al16(dw_vocab)))
    return set_error(FL_ERR_ALIGN, "h / w / dh / dw not 16-byte aligned");
  if (!std::isfinite(grad_scale)) return set_error(FL_ERR_ARG, "grad_scale is not finite");
  const long V = c->d.vocab, H = c->d.hidden;
  if (overlap(dh, T * H * c->E, h, T * H * c->E) || overlap(dh, T * H * c->E, workspace, workspace_bytes))
    return set_error(FL_ERR_ALIAS, "dh overlaps h / the workspace");
  if (dw_vocab && (overlap(dw_vocab, V * H * 4, workspace, workspace_bytes) ||
                   overlap(dw_vocab, V * H * 4, dh, T * H * c->E)))
    return set_error(FL_ERR_ALIAS, "dw overlaps dh / the workspace");
  const ClientWs w = carve(c, T, (char*)workspace);
  hipStream_t s = (hipStream_t)stream;
  if (c->d.dtype == FL_BF16)
    hipLaunchKernelGGL(ce_bwd_kernel<bf16>, dim3((unsigned)T), dim3(kThreads), 0, s, (bf16*)w.logits, c->vpad,
                       (int)V, w.labels, w.lse, grad_scale);
  else
    hipLaunchKernelGGL(ce_bwd_kernel<float>, dim3((unsigned)T), dim3(kThreads), 0, s, (float*)w.logits, c->vpad,
                       (int)V, w.labels, w.lse, grad_scale);
  CK(hipGetLastError());
  // dh = dlogits W   (reduction over the padded vocabulary; W's rows past V
  // read as zero); with the final LayerNorm this is the gradient at its output
  GemmDesc g;
  g.A = w.logits; g.B = w_vocab; g.C = ln_g ? (void*)w.dhn : dh;
  g.M = (int)T; g.N = (int)H; g.K = (int)c->vpad;
  g.lda = c->vpad; g.ldb = H; g.ldc = H;
  g.b_rows = (int)V;
  g.part = w.part; g.part_bytes = w.part_bytes;
  CK(gemm(dt_of(c), GEMM_NN, EPI_STORE, g, s));
  if (ln_g) {
    CK(layernorm_bwd_dx(dt_of(c), w.dhn, h, w.mean, w.rstd, ln_g, nullptr, dh, (int)T, (int)H, s));
    if (dln_g) {
      const int nb = colsum_blocks((int)T);
      CK(colsum_partial(dt_of(c), 1, w.dhn, H, h, w.mean, w.rstd, (int)T, (int)H, w.ln_part, w.ln_part2, s));
      CK(colsum_finish(w.ln_part, nb, (int)H, dln_g, s));
      CK(colsum_finish(w.ln_part2, nb, (int)H, dln_b, s));
    }
  }
  if (!dw_vocab) return FL_OK;
  // dW += dlogits^T hn   (rows m < V of the padded logits' columns; hn = h
  // without the final LayerNorm)
  GemmDesc gw;
  gw.A = w.logits; gw.B = ln_g ? (const void*)w.hn : h; gw.C = dw_vocab;
  gw.M = (int)V; gw.N = (int)H; gw.K = (int)T;
  gw.lda = c->vpad; gw.ldb = H; gw.ldc = H;
  gw.part = w.part; gw.part_bytes = w.part_bytes;
  CK(gemm(dt_of(c), GEMM_TN, EPI_ACC_F32, gw, s));
  return FL_OK;
}

}  // extern "C"
