// The server-stack engine behind the C ABI: descriptor validation, memory
// plan (saved activations and workspace carving), batch-plan upload, and the
// per-block kernel sequence of the forward and backward passes, all enqueued
// on the caller's stream with no host synchronisation.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "../../include/flglm.h"
#include "kernels.h"

using namespace flglm;

namespace {

thread_local std::string g_err;

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

#define HIP_OK(expr)                                                                      \
  do {                                                                                    \
    hipError_t e_ = (expr);                                                               \
    if (e_ != hipSuccess) return fail(FL_ERR_HIP, "%s: %s", #expr, hipGetErrorString(e_)); \
  } while (0)

// Enqueue one launch (an expression returning hipError_t) with its algorithmic
// flops and bytes; timed when profiling is on.  Needs `st` and `s` in scope.
#define LAUNCH(cls, flops, bytes, ...) \
  HIP_OK(timed(st, s, (cls), (flops), (bytes), [&]() { return (__VA_ARGS__); }))

constexpr size_t kAlign = 256;
inline size_t align_up(size_t v) { return (v + kAlign - 1) / kAlign * kAlign; }

// Bump allocator over a caller-provided region (or a dry run for sizing).
struct Carver {
  char* base;
  size_t off = 0;
  explicit Carver(void* b) : base(static_cast<char*>(b)) {}
  void* take(size_t bytes) {
    void* p = base ? base + off : nullptr;
    off += align_up(bytes);
    return p;
  }
};

// Per-block forward intermediates.
struct Acts {
  void *u, *qkv, *o, *h, *w, *z, *g;
  float *lse, *mean1, *rstd1, *mean2, *rstd2;
};

}  // namespace

struct fl_stack {
  fl_stack_desc d;
  int E;   // element bytes
  int hd;  // head dim
  static constexpr int kRing = 4;
  void* stage[kRing] = {};
  size_t stage_cap[kRing] = {};
  hipEvent_t ev[kRing] = {};
  bool ev_made[kRing] = {};
  bool ev_used[kRing] = {};
  int next = 0;
  // opt-in launch timing (fl_stack_profile)
  struct Rec {
    int cls;
    hipEvent_t a, b;
    double flops, bytes;
  };
  uint32_t prof_mask = 0;  // bit c: launches of class c are timed
  std::vector<Rec> recs;
  std::vector<hipEvent_t> pool;
};


namespace {

const char* const kProfNames[FL_PROF_NUM_CLASSES] = {
    "plan",          "layernorm_fwd", "gemm_nt_bias", "rope_qk",  "attn_fwd",     "gemm_nt_bias_res", "gemm_nt_bias_gelu",
    "gemm_tn_acc",   "gemm_nn_gelu_bwd", "gemm_nn",   "layernorm_bwd", "colsum", "attn_bwd", "prefix_grad"};

hipError_t take_event(fl_stack* st, hipEvent_t* e) {
  if (!st->pool.empty()) {
    *e = st->pool.back();
    st->pool.pop_back();
    return hipSuccess;
  }
  return hipEventCreate(e);
}

// Runs `launch` (returning hipError_t); when profiling is on, brackets it
// with two events on stream s and records the launch's algorithmic work.
template <class Fn>
hipError_t timed(fl_stack* st, hipStream_t s, int cls, double flops, double bytes, Fn&& launch) {
  if (!((st->prof_mask >> cls) & 1u)) return launch();
  fl_stack::Rec r{cls, nullptr, nullptr, flops, bytes};
  hipError_t e = take_event(st, &r.a);
  if (e != hipSuccess) return e;
  if ((e = take_event(st, &r.b)) != hipSuccess) {
    st->pool.push_back(r.a);
    return e;
  }
  if ((e = hipEventRecord(r.a, s)) != hipSuccess) {
    st->pool.push_back(r.a);
    st->pool.push_back(r.b);
    return e;
  }
  e = launch();
  hipError_t e2 = hipEventRecord(r.b, s);
  st->recs.push_back(r);
  return e != hipSuccess ? e : e2;
}

}  // namespace

namespace {

struct BatchInfo {
  int T, S, C, maxL;
  bool prefix;
  double pairs;  // sum over sequences of visible (query, key) pairs
  // the descriptor's host sequence bounds (valid during the call)
  const int32_t* cu_host;
  const int32_t* prefix_host;
};

int validate_batch(const fl_batch_desc* b, BatchInfo* bi) {
  if (!b) return fail(FL_ERR_NULL, "batch descriptor is NULL");
  if (!b->cu_seqlens || !b->client_seq_ptr) return fail(FL_ERR_NULL, "cu_seqlens / client_seq_ptr is NULL");
  if (b->num_seqs < 1) return fail(FL_ERR_SEQLENS, "num_seqs must be >= 1 (got %d)", b->num_seqs);
  if (b->num_clients < 1) return fail(FL_ERR_CLIENTS, "num_clients must be >= 1 (got %d)", b->num_clients);
  if (b->num_clients > b->num_seqs)
    return fail(FL_ERR_CLIENTS, "num_clients %d > num_seqs %d", b->num_clients, b->num_seqs);
  if (b->total_tokens < 1 || b->total_tokens > (int64_t)(1 << 26))
    return fail(FL_ERR_SEQLENS, "total_tokens %lld out of range [1, 2^26]", (long long)b->total_tokens);
  const int32_t* cu = b->cu_seqlens;
  if (cu[0] != 0) return fail(FL_ERR_SEQLENS, "cu_seqlens[0] must be 0");
  int maxL = 0;
  for (int s = 0; s < b->num_seqs; ++s) {
    const int L = cu[s + 1] - cu[s];
    if (L < 1) return fail(FL_ERR_SEQLENS, "sequence %d has length %d (must be >= 1)", s, L);
    maxL = std::max(maxL, L);
  }
  if ((int64_t)cu[b->num_seqs] != b->total_tokens)
    return fail(FL_ERR_SEQLENS, "cu_seqlens[S] = %d != total_tokens %lld", cu[b->num_seqs],
                (long long)b->total_tokens);
  if (b->max_seqlen != maxL) return fail(FL_ERR_SEQLENS, "max_seqlen %d != longest sequence %d", b->max_seqlen, maxL);
  const int32_t* csp = b->client_seq_ptr;
  if (csp[0] != 0) return fail(FL_ERR_CLIENTS, "client_seq_ptr[0] must be 0");
  for (int c = 0; c < b->num_clients; ++c)
    if (csp[c + 1] <= csp[c]) return fail(FL_ERR_CLIENTS, "client %d owns no sequences", c);
  if (csp[b->num_clients] != b->num_seqs)
    return fail(FL_ERR_CLIENTS, "client_seq_ptr[C] = %d != num_seqs %d", csp[b->num_clients], b->num_seqs);
  if (b->mask_kind != FL_MASK_CAUSAL && b->mask_kind != FL_MASK_PREFIX)
    return fail(FL_ERR_PREFIX, "unknown mask_kind %d", b->mask_kind);
  if (b->mask_kind == FL_MASK_PREFIX) {
    if (!b->prefix_len) return fail(FL_ERR_NULL, "prefix_len is NULL with FL_MASK_PREFIX");
    for (int s = 0; s < b->num_seqs; ++s) {
      const int L = cu[s + 1] - cu[s];
      if (b->prefix_len[s] < 0 || b->prefix_len[s] > L)
        return fail(FL_ERR_PREFIX, "prefix_len[%d] = %d outside [0, %d]", s, b->prefix_len[s], L);
    }
  }
  bi->T = (int)b->total_tokens;
  bi->S = b->num_seqs;
  bi->C = b->num_clients;
  bi->maxL = maxL;
  bi->prefix = b->mask_kind == FL_MASK_PREFIX;
  bi->cu_host = cu;
  bi->prefix_host = bi->prefix ? b->prefix_len : nullptr;
  bi->pairs = 0;
  for (int s = 0; s < b->num_seqs; ++s) {
    const double L = cu[s + 1] - cu[s];
    const double P = bi->prefix ? b->prefix_len[s] : 0;
    // causal pairs L(L+1)/2, plus the pairs a bidirectional prefix adds
    bi->pairs += L * (L + 1) / 2 + (P > 1 ? P * (P - 1) / 2 : 0);
  }
  return FL_OK;
}

int validate_desc(const fl_stack_desc* d) {
  if (!d) return fail(FL_ERR_NULL, "stack descriptor is NULL");
  if (d->dtype != FL_BF16 && d->dtype != FL_F32) return fail(FL_ERR_SHAPE, "unknown dtype %d", d->dtype);
  if (d->num_layers < 1) return fail(FL_ERR_SHAPE, "num_layers must be >= 1");
  if (d->hidden < 256 || d->hidden % 256 != 0 || d->hidden > 4096)
    return fail(FL_ERR_SHAPE, "hidden %d must be a multiple of 256 in [256, 4096]", d->hidden);
  if (d->num_heads < 1 || d->hidden % d->num_heads != 0) return fail(FL_ERR_SHAPE, "hidden %% num_heads != 0");
  const int hd = d->hidden / d->num_heads;
  if (hd != 64 && hd != 128) return fail(FL_ERR_SHAPE, "head dim %d not in {64, 128}", hd);
  if (d->ffn_hidden < 256 || d->ffn_hidden % 256 != 0)
    return fail(FL_ERR_SHAPE, "ffn_hidden %d must be a positive multiple of 256", d->ffn_hidden);
  if (d->rotary_dim < 0 || d->rotary_dim > hd || d->rotary_dim % 32 != 0)
    return fail(FL_ERR_SHAPE, "rotary_dim %d must be a multiple of 32 in [0, head dim]", d->rotary_dim);
  if (!(d->rope_base > 0.f)) return fail(FL_ERR_SHAPE, "rope_base must be > 0");
  if (!(d->ln_eps > 0.f)) return fail(FL_ERR_SHAPE, "ln_eps must be > 0");
  if (d->num_prefix < 0 || d->num_prefix > 4096)
    return fail(FL_ERR_SHAPE, "num_prefix %d must be in [0, 4096]", d->num_prefix);
  if (d->num_prefix > 0 && d->dtype != FL_BF16)
    return fail(FL_ERR_SHAPE, "the P-tuning v2 prefix (num_prefix > 0) needs dtype FL_BF16");
  if (!(d->residual_alpha >= 0.f) || !std::isfinite(d->residual_alpha))
    return fail(FL_ERR_SHAPE, "residual_alpha must be finite and >= 0");
  if (d->rotary_2d != 0 && d->rotary_2d != 1) return fail(FL_ERR_SHAPE, "rotary_2d must be 0 or 1");
  if (d->rotary_2d && 2 * d->rotary_dim != hd)
    return fail(FL_ERR_SHAPE, "GLM 2-D positions need rotary_dim = head dim / 2");
  return FL_OK;
}

// ---------------------------------------------------------------------------
// Memory plan
// ---------------------------------------------------------------------------
struct Plan {
  int32_t* cu;
  int32_t* prefix;
  int32_t* pos;
  int32_t* pos2;  // GLM block positions (2-D mode)
  float* cos_t;
  float* sin_t;
  float* gemm_part;  // split-reduction scratch of the bf16 GEMMs (null for fp32)
  size_t gemm_part_bytes;
};

void carve_plan(Carver& cv, const BatchInfo& bi, int rotary_dim, Plan* p) {
  p->cu = (int32_t*)cv.take(sizeof(int32_t) * (bi.S + 1));
  p->prefix = (int32_t*)cv.take(sizeof(int32_t) * bi.S);
  p->pos = (int32_t*)cv.take(sizeof(int32_t) * bi.T);
  p->pos2 = (int32_t*)cv.take(sizeof(int32_t) * bi.T);
  // positions 0..maxL (a GLM block position reaches L when the context is empty)
  const size_t tab = sizeof(float) * (size_t)(bi.maxL + 1) * std::max(rotary_dim / 2, 1);
  p->cos_t = (float*)cv.take(tab);
  p->sin_t = (float*)cv.take(tab);
}

// with_z = false: no room for the FFN pre-activation (an inference forward
// never stores it).
void carve_acts(Carver& cv, const fl_stack* st, int T, Acts* a, bool with_z = true) {
  const size_t E = st->E, H = st->d.hidden, F = st->d.ffn_hidden, nh = st->d.num_heads;
  a->u = cv.take(E * T * H);
  a->qkv = cv.take(E * T * 3 * H);
  a->o = cv.take(E * T * H);
  a->h = cv.take(E * T * H);
  a->w = cv.take(E * T * H);
  a->z = with_z ? cv.take(E * T * F) : nullptr;
  a->g = cv.take(E * T * F);
  a->lse = (float*)cv.take(sizeof(float) * T * nh);
  a->mean1 = (float*)cv.take(sizeof(float) * T);
  a->rstd1 = (float*)cv.take(sizeof(float) * T);
  a->mean2 = (float*)cv.take(sizeof(float) * T);
  a->rstd2 = (float*)cv.take(sizeof(float) * T);
}

// saved = [acts_0 .. acts_{N-1}] (recompute == 0), then x_1 .. x_{N-1}.
struct Saved {
  std::vector<Acts> acts;
  std::vector<void*> xin;  // xin[l] = input of block l (xin[0] unused: the caller's x)
};
void carve_saved(Carver& cv, const fl_stack* st, int T, bool recompute, Saved* s) {
  const int N = st->d.num_layers;
  s->acts.assign(N, Acts{});
  s->xin.assign(N, nullptr);
  if (!recompute)
    for (int l = 0; l < N; ++l) carve_acts(cv, st, T, &s->acts[l]);
  for (int l = 1; l < N; ++l) s->xin[l] = cv.take((size_t)st->E * T * st->d.hidden);
}

struct Work {
  Plan plan;
  Acts acts;      // forward intermediates when not saved / recomputed in backward
  void* ping[2];  // block outputs (inference) / gradient ping-pong (backward)
  void *dz, *dh, *tmp, *dqkv;
  float* delta;
  float *part, *part2;
  float* lnp[3];  // fused LayerNorm backward partials: gain, shift, output sums, [kLnBlocks][H] each
  float* dprefix;
  // stored attention softmax gradient (bf16, see attn_ds_tiles) and its
  // per-sequence offsets; null above kAttnDsMaxBytes (dq then recomputes it)
  void* ds;
  int64_t* ds_off;
  // with ds: b_qkv's column sums per 64-row tile of each sequence, formed by
  // the attention backward (bias_rows x 3H fp32) and its tile table
  float* bias_part;
  int32_t* tile_base;
  int bias_rows;
};
// The stored softmax gradient grows with the sum of squared sequence
// lengths (about 1.9 GB for 32 heads over 32 sequences of 512 to 2048
// tokens); beyond this, the backward recomputes it in the dq kernel.
constexpr size_t kAttnDsMaxBytes = size_t(8) << 30;
void carve_work(Carver& cv, const fl_stack* st, const BatchInfo& bi, Work* w) {
  const size_t E = st->E, H = st->d.hidden, F = st->d.ffn_hidden, T = bi.T;
  carve_plan(cv, bi, st->d.rotary_dim, &w->plan);
  w->plan.gemm_part_bytes = st->d.dtype == FL_BF16 ? gemm_part_bytes() : 0;
  w->plan.gemm_part = w->plan.gemm_part_bytes ? (float*)cv.take(w->plan.gemm_part_bytes) : nullptr;
  carve_acts(cv, st, bi.T, &w->acts);
  w->ping[0] = cv.take(E * T * H);
  w->ping[1] = cv.take(E * T * H);
  w->dz = cv.take(E * T * F);
  w->dh = cv.take(E * T * H);
  w->tmp = cv.take(E * T * H);
  w->dqkv = cv.take(E * T * 3 * H);
  w->delta = (float*)cv.take(sizeof(float) * T * st->d.num_heads);
  const size_t nmax = std::max(F, 3 * H);
  w->part = (float*)cv.take(sizeof(float) * colsum_blocks(bi.T) * nmax);
  w->part2 = (float*)cv.take(sizeof(float) * colsum_blocks(bi.T) * nmax);
  for (int i = 0; i < 3; ++i) w->lnp[i] = (float*)cv.take(sizeof(float) * kLnBlocks * H);
  // per-sequence P-tuning v2 prefix gradients, [2][S][L_p][H] fp32
  const size_t np = st->d.num_prefix;
  w->dprefix = np ? (float*)cv.take(sizeof(float) * 2 * bi.S * np * H) : nullptr;
  w->ds = nullptr;
  w->ds_off = nullptr;
  w->bias_part = nullptr;
  w->tile_base = nullptr;
  w->bias_rows = 0;
  if (st->d.dtype == FL_BF16) {
    const size_t ds_bytes =
        attn_ds_tiles(bi.cu_host, bi.prefix_host, bi.S, st->d.num_heads, st->d.num_prefix) * kAttnDsTileBytes;
    if (ds_bytes <= kAttnDsMaxBytes) {
      w->ds_off = (int64_t*)cv.take(attn_ds_off_bytes(bi.S));
      w->ds = cv.take(ds_bytes);
      int rows = 0;
      for (int q = 0; q < bi.S; ++q) rows += (bi.cu_host[q + 1] - bi.cu_host[q] + 63) / 64;
      w->bias_rows = rows;
      w->tile_base = (int32_t*)cv.take(sizeof(int32_t) * (bi.S + 1));
      w->bias_part = (float*)cv.take(sizeof(float) * (size_t)rows * 3 * H);
    }
  }
}

size_t saved_bytes(const fl_stack* st, const BatchInfo& bi, bool recompute) {
  Carver cv(nullptr);
  Saved s;
  carve_saved(cv, st, bi.T, recompute, &s);
  return cv.off;
}
size_t work_bytes(const fl_stack* st, const BatchInfo& bi) {
  Carver cv(nullptr);
  Work w;
  carve_work(cv, st, bi, &w);
  return cv.off;
}

// What an inference forward (no saved activations) touches: the batch plan,
// the GEMM split-reduction scratch, one block's intermediates without z,
// and the two ping-pong block outputs.  Same sizes as carve_work's, so the
// GEMMs split their reductions the same way.
void carve_fwd_work(Carver& cv, const fl_stack* st, const BatchInfo& bi, Work* w) {
  const size_t E = st->E, H = st->d.hidden, T = bi.T;
  *w = Work();
  carve_plan(cv, bi, st->d.rotary_dim, &w->plan);
  w->plan.gemm_part_bytes = st->d.dtype == FL_BF16 ? gemm_part_bytes() : 0;
  w->plan.gemm_part = w->plan.gemm_part_bytes ? (float*)cv.take(w->plan.gemm_part_bytes) : nullptr;
  carve_acts(cv, st, bi.T, &w->acts, false);
  w->ping[0] = cv.take(E * T * H);
  w->ping[1] = cv.take(E * T * H);
}
size_t fwd_work_bytes(const fl_stack* st, const BatchInfo& bi) {
  Carver cv(nullptr);
  Work w;
  carve_fwd_work(cv, st, bi, &w);
  return cv.off;
}

// ---------------------------------------------------------------------------
// Checks on device pointers
// ---------------------------------------------------------------------------
bool aligned16(const void* p) { return ((uintptr_t)p & 15) == 0; }
bool overlap(const void* a, size_t na, const void* b, size_t nb) {
  if (!a || !b || na == 0 || nb == 0) return false;
  uintptr_t x = (uintptr_t)a, y = (uintptr_t)b;
  return x < y + nb && y < x + na;
}

int check_params(const fl_stack* st, const fl_layer_params* layers) {
  if (!layers) return fail(FL_ERR_NULL, "layers is NULL");
  const int n = st->d.num_prefix ? 14 : 12;
  for (int l = 0; l < st->d.num_layers; ++l) {
    const void* ps[14] = {layers[l].w_qkv, layers[l].b_qkv, layers[l].w_o,   layers[l].b_o,   layers[l].w_1,
                          layers[l].b_1,   layers[l].w_2,   layers[l].b_2,   layers[l].ln1_g, layers[l].ln1_b,
                          layers[l].ln2_g, layers[l].ln2_b, layers[l].prefix_k, layers[l].prefix_v};
    for (int i = 0; i < n; ++i) {
      if (!ps[i]) return fail(FL_ERR_NULL, "layer %d parameter %d is NULL", l, i);
      if (!aligned16(ps[i])) return fail(FL_ERR_ALIGN, "layer %d parameter %d is not 16-byte aligned", l, i);
    }
  }
  return FL_OK;
}

// Weight gradients: all twelve set (trained) or all NULL (frozen).  Prefix
// gradients: required with a prefix.
int check_grads(const fl_stack* st, const fl_layer_grads* grads) {
  if (!grads) return fail(FL_ERR_NULL, "grads is NULL");
  for (int l = 0; l < st->d.num_layers; ++l) {
    const float* ps[12] = {grads[l].w_qkv, grads[l].b_qkv, grads[l].w_o, grads[l].b_o,
                           grads[l].w_1,   grads[l].b_1,   grads[l].w_2, grads[l].b_2,
                           grads[l].ln1_g, grads[l].ln1_b, grads[l].ln2_g, grads[l].ln2_b};
    const bool frozen = ps[0] == nullptr;
    for (int i = 0; i < 12; ++i) {
      if (frozen != (ps[i] == nullptr))
        return fail(FL_ERR_NULL, "layer %d: weight gradients must be all set or all NULL (gradient %d)", l, i);
      if (ps[i] && !aligned16(ps[i])) return fail(FL_ERR_ALIGN, "layer %d gradient %d is not 16-byte aligned", l, i);
    }
    if (st->d.num_prefix) {
      if (!grads[l].prefix_k || !grads[l].prefix_v)
        return fail(FL_ERR_NULL, "layer %d: prefix gradients are NULL with num_prefix > 0", l);
      if (!aligned16(grads[l].prefix_k) || !aligned16(grads[l].prefix_v))
        return fail(FL_ERR_ALIGN, "layer %d prefix gradient is not 16-byte aligned", l);
    }
  }
  return FL_OK;
}

// ---------------------------------------------------------------------------
// Plan upload: host descriptor arrays -> pinned staging ring -> workspace.
// ---------------------------------------------------------------------------
// Once cu_seqlens and the prefix lengths are on the device: every row's
// position inside its sequence and the rotary table.
int plan_kernels(fl_stack* st, const BatchInfo& bi, const Plan& p, hipStream_t stream) {
  hipStream_t s = stream;
  LAUNCH(FL_PROF_PLAN, 0, 4.0 * bi.T, [&]() {
    hipError_t e = st->d.rotary_2d ? seq_positions_2d(p.cu, bi.prefix ? p.prefix : nullptr, bi.S, p.pos, p.pos2, stream)
                                   : seq_positions(p.cu, bi.S, p.pos, stream);
    return e != hipSuccess ? e
                           : rope_table(p.cos_t, p.sin_t, bi.maxL + 1, st->d.rotary_dim, st->d.rope_base, stream);
  }());
  return FL_OK;
}

int upload_plan(fl_stack* st, const fl_batch_desc* b, const BatchInfo& bi, const Plan& p, hipStream_t stream) {
  const size_t ncu = bi.S + 1, npre = bi.S;
  const size_t bytes = sizeof(int32_t) * (ncu + npre);
  const int k = st->next;
  st->next = (st->next + 1) % fl_stack::kRing;
  if (!st->ev_made[k]) {
    HIP_OK(hipEventCreateWithFlags(&st->ev[k], hipEventDisableTiming));
    st->ev_made[k] = true;
  }
  if (st->ev_used[k]) HIP_OK(hipEventSynchronize(st->ev[k]));
  if (st->stage_cap[k] < bytes) {
    if (st->stage[k]) HIP_OK(hipHostFree(st->stage[k]));
    st->stage[k] = nullptr;
    st->stage_cap[k] = 0;
    HIP_OK(hipHostMalloc(&st->stage[k], std::max(bytes, (size_t)4096), hipHostMallocDefault));
    st->stage_cap[k] = std::max(bytes, (size_t)4096);
  }
  int32_t* h = (int32_t*)st->stage[k];
  std::memcpy(h, b->cu_seqlens, sizeof(int32_t) * ncu);
  if (bi.prefix) std::memcpy(h + ncu, b->prefix_len, sizeof(int32_t) * npre);
  else std::memset(h + ncu, 0, sizeof(int32_t) * npre);
  HIP_OK(hipMemcpyAsync(p.cu, h, sizeof(int32_t) * ncu, hipMemcpyHostToDevice, stream));
  HIP_OK(hipMemcpyAsync(p.prefix, h + ncu, sizeof(int32_t) * npre, hipMemcpyHostToDevice, stream));
  HIP_OK(hipEventRecord(st->ev[k], stream));
  st->ev_used[k] = true;
  return plan_kernels(st, bi, p, stream);
}

// Algorithmic work of one launch, for the opt-in launch timing.
double gemm_flops(double M, double N, double K) { return 2.0 * M * N * K; }
double gemm_bytes(double M, double N, double K, double E, double Eout) { return (M * K + N * K) * E + M * N * Eout; }

// ---------------------------------------------------------------------------
// One block forward.  `out` may be NULL (recompute for the backward: the
// final projection is not needed).
// ---------------------------------------------------------------------------
// Hands the GEMM the workspace's split-reduction scratch.
GemmDesc& with_part(GemmDesc& g, const Plan& plan) {
  g.part = plan.gemm_part;
  g.part_bytes = plan.gemm_part_bytes;
  return g;
}

// keep_z = false: the FFN's pre-activation z is not stored (nothing reads it
// when the block's intermediates are not kept for a backward).
int block_forward(fl_stack* st, const BatchInfo& bi, const Plan& plan, const fl_layer_params& p, const void* x,
                  const Acts& a, void* out, hipStream_t s, bool keep_z = true) {
  const DType dt = (DType)st->d.dtype;
  const int T = bi.T, H = st->d.hidden, F = st->d.ffn_hidden;
  const double E = st->E, TH = (double)T * H;
  LAUNCH(FL_PROF_LAYERNORM_FWD, 0, 2 * TH * E + 8.0 * T,
         layernorm_fwd(dt, x, p.ln1_g, p.ln1_b, a.u, a.mean1, a.rstd1, T, H, st->d.ln_eps, s));
  GemmDesc g;
  g.A = a.u; g.B = p.w_qkv; g.C = a.qkv; g.M = T; g.N = 3 * H; g.K = H;
  g.lda = H; g.ldb = H; g.ldc = 3 * H; g.bias = p.b_qkv;
  LAUNCH(FL_PROF_GEMM_NT_BIAS, gemm_flops(T, 3 * H, H), gemm_bytes(T, 3 * H, H, E, E),
         gemm(dt, GEMM_NT, EPI_BIAS, with_part(g, plan), s));
  // q and k: the first rotary_dim features of every head, read and written.
  // A separate pass on purpose: folded into the QKV epilogue (a lane-pair
  // exchange plus table loads per row) it measured 0.5 ms slower per call
  // at T = 41447 than this 0.14 ms kernel, the epilogue being latency-bound.
  // (GLM 2-D positions: the second half by the block position, same pass)
  const int32_t* pos2 = st->d.rotary_2d ? plan.pos2 : nullptr;
  LAUNCH(FL_PROF_ROPE, 0, 4.0 * T * st->d.num_heads * st->d.rotary_dim * E * (pos2 ? 2 : 1),
         rope_qk(dt, a.qkv, 3 * H, plan.pos, plan.cos_t, plan.sin_t, T, H, st->hd, st->d.rotary_dim, s, 1.f, pos2));
  const float alpha = st->d.residual_alpha;
  AttnDesc ad;
  ad.qkv = a.qkv; ad.ld_qkv = 3 * H; ad.o = a.o; ad.ld_o = H; ad.lse = a.lse;
  ad.cu_seqlens = plan.cu; ad.prefix_len = bi.prefix ? plan.prefix : nullptr;
  ad.num_seqs = bi.S; ad.max_seqlen = bi.maxL; ad.num_heads = st->d.num_heads; ad.head_dim = st->hd;
  ad.hidden = H; ad.total_tokens = T;
  ad.pk = p.prefix_k; ad.pv = p.prefix_v; ad.num_prefix = st->d.num_prefix;
  const double pairs = bi.pairs + (double)st->d.num_prefix * T;  // every query sees the whole prefix
  LAUNCH(FL_PROF_ATTN_FWD, 4.0 * H * pairs, 4 * TH * E + 4.0 * T * st->d.num_heads, attn_fwd(dt, ad, s));
  g = GemmDesc();
  g.A = a.o; g.B = p.w_o; g.C = a.h; g.M = T; g.N = H; g.K = H;
  g.lda = H; g.ldb = H; g.ldc = H; g.bias = p.b_o; g.ldr = H;
  g.R = alpha > 0.f ? a.u : x;  // ChatGLM-6B: h = alpha u + ...
  g.res_scale = alpha > 0.f ? alpha : 1.f;
  LAUNCH(FL_PROF_GEMM_NT_BIAS_RES, gemm_flops(T, H, H), gemm_bytes(T, H, H, E, E) + TH * E,
         gemm(dt, GEMM_NT, EPI_BIAS_RES, with_part(g, plan), s));
  LAUNCH(FL_PROF_LAYERNORM_FWD, 0, 2 * TH * E + 8.0 * T,
         layernorm_fwd(dt, a.h, p.ln2_g, p.ln2_b, a.w, a.mean2, a.rstd2, T, H, st->d.ln_eps, s));
  g = GemmDesc();
  g.A = a.w; g.B = p.w_1; g.C = keep_z ? a.z : nullptr; g.C2 = a.g; g.M = T; g.N = F; g.K = H;
  g.lda = H; g.ldb = H; g.ldc = F; g.ldc2 = F; g.bias = p.b_1;
  LAUNCH(FL_PROF_GEMM_NT_BIAS_GELU, gemm_flops(T, F, H), gemm_bytes(T, F, H, E, keep_z ? 2 * E : E),
         gemm(dt, GEMM_NT, EPI_BIAS_GELU, with_part(g, plan), s));
  if (out) {
    g = GemmDesc();
    g.A = a.g; g.B = p.w_2; g.C = out; g.M = T; g.N = H; g.K = F;
    g.lda = F; g.ldb = F; g.ldc = H; g.bias = p.b_2; g.ldr = H;
    g.R = alpha > 0.f ? a.w : a.h;  // ChatGLM-6B: y = alpha w + ...
    g.res_scale = alpha > 0.f ? alpha : 1.f;
    LAUNCH(FL_PROF_GEMM_NT_BIAS_RES, gemm_flops(T, H, F), gemm_bytes(T, H, F, E, E) + TH * E,
           gemm(dt, GEMM_NT, EPI_BIAS_RES, with_part(g, plan), s));
  }
  return FL_OK;
}

// out[n] += sum_t X[t][n] (two-stage, deterministic).
int colsum_into(fl_stack* st, DType dt, const void* X, long ldx, int T, int N, float* out, const Work& w,
                hipStream_t s) {
  LAUNCH(FL_PROF_COLSUM, 0, (double)T * N * st->E, [&]() {
    hipError_t e = colsum_partial(dt, 0, X, ldx, nullptr, nullptr, nullptr, T, N, w.part, nullptr, s);
    return e != hipSuccess ? e : colsum_finish(w.part, colsum_blocks(T), N, out, s);
  }());
  return FL_OK;
}

// LayerNorm backward: dx = dres + LN^T(dy); gain / shift gradients (NULL:
// frozen) += their column sums and, with dsum, dsum += the column sums of dx
// (the bias gradient of the projection that produced the LayerNorm's
// input), all in the one pass over dy and x.
int ln_backward(fl_stack* st, DType dt, const void* dy, const void* xin, const float* mean, const float* rstd,
                const void* gamma, const void* dres, void* dx, float* dgamma, float* dbeta, float* dsum, int T, int H,
                const Work& w, hipStream_t s) {
  const double TH = (double)T * H, E = st->E;
  LAUNCH(FL_PROF_LAYERNORM_BWD, 0, (dres ? 4 : 3) * TH * E + 8.0 * T,
         layernorm_bwd_fused(dt, dy, xin, mean, rstd, gamma, dres, dx, T, H, dgamma ? w.lnp[0] : nullptr,
                             dgamma ? w.lnp[1] : nullptr, dsum ? w.lnp[2] : nullptr, s));
  if (!dgamma && !dsum) return FL_OK;
  LAUNCH(FL_PROF_COLSUM, 0, 4.0 * kLnBlocks * H * ((dgamma ? 2 : 0) + (dsum ? 1 : 0)), [&]() {
    const float* parts[3];
    float* outs[3];
    int n = 0;
    if (dgamma) {
      parts[n] = w.lnp[0]; outs[n++] = dgamma;
      parts[n] = w.lnp[1]; outs[n++] = dbeta;
    }
    if (dsum) { parts[n] = w.lnp[2]; outs[n++] = dsum; }
    return colsum_finish_n(parts, outs, n, kLnBlocks, H, s);
  }());
  return FL_OK;
}

// One block backward: dy -> dx, gradients += .
// dx_sum (or NULL): receives += the column sums of dx, formed in the last
// LayerNorm backward's pass (dx is the dy of the block below, whose bias
// gradient db_2 is that sum); b2_done: this block's db_2 was already added
// that way by the block above.
int block_backward(fl_stack* st, const BatchInfo& bi, const Plan& plan, const Work& w, const fl_layer_params& p,
                   const fl_layer_grads& gr, const void* x, const Acts& a, const void* dy, void* dx, hipStream_t s,
                   float* dx_sum, bool b2_done) {
  const DType dt = (DType)st->d.dtype;
  const int T = bi.T, H = st->d.hidden, F = st->d.ffn_hidden;
  const double E = st->E;
  // frozen weights (P-tuning v2): input gradients and prefix gradients only
  const bool train_w = gr.w_qkv != nullptr;
  // ChatGLM-6B's residual: the normalised inputs w and u, scaled by alpha,
  // feed y and h, so dy and dh join the LayerNorm inputs' gradients (in the
  // input-gradient GEMMs' epilogues) instead of passing straight through
  const float alpha = st->d.residual_alpha;
  int rc;
  // y = h + g W_2^T + b_2
  GemmDesc g;
  if (train_w) {
    if (!b2_done && (rc = colsum_into(st, dt, dy, H, T, H, gr.b_2, w, s))) return rc;
    g.A = dy; g.B = a.g; g.C = gr.w_2; g.M = H; g.N = F; g.K = T; g.lda = H; g.ldb = F; g.ldc = F;
    LAUNCH(FL_PROF_GEMM_TN_ACC, gemm_flops(H, F, T), gemm_bytes(H, F, T, E, 8),
           gemm(dt, GEMM_TN, EPI_ACC_F32, with_part(g, plan), s));
  }
  g = GemmDesc();
  g.A = dy; g.B = p.w_2; g.C = w.dz; g.M = T; g.N = F; g.K = H; g.lda = H; g.ldb = F; g.ldc = F;
  g.Z = a.z; g.ldz = F;
  // db_1 = column sums of dz: formed per 256-row tile in the GEMM's epilogue
  // where the kernel supports it (no second pass over dz), else below
  const bool b1_fused = train_w && gemm_fuses_colsum(dt, GEMM_NN, EPI_GELU_BWD, g);
  if (b1_fused) g.colsum = w.part;
  LAUNCH(FL_PROF_GEMM_NN_GELU_BWD, gemm_flops(T, F, H), gemm_bytes(T, F, H, E, 2 * E),
         gemm(dt, GEMM_NN, EPI_GELU_BWD, with_part(g, plan), s));
  // z = w W_1^T + b_1
  if (train_w) {
    if (b1_fused) {
      LAUNCH(FL_PROF_COLSUM, 0, 4.0 * colsum_blocks(T) * F, colsum_finish(w.part, colsum_blocks(T), F, gr.b_1, s));
    } else if ((rc = colsum_into(st, dt, w.dz, F, T, F, gr.b_1, w, s))) {
      return rc;
    }
    g = GemmDesc();
    g.A = w.dz; g.B = a.w; g.C = gr.w_1; g.M = F; g.N = H; g.K = T; g.lda = F; g.ldb = H; g.ldc = H;
    LAUNCH(FL_PROF_GEMM_TN_ACC, gemm_flops(F, H, T), gemm_bytes(F, H, T, E, 8),
           gemm(dt, GEMM_TN, EPI_ACC_F32, with_part(g, plan), s));
  }
  g = GemmDesc();
  g.A = w.dz; g.B = p.w_1; g.C = w.tmp; g.M = T; g.N = H; g.K = F; g.lda = F; g.ldb = H; g.ldc = H;
  if (alpha > 0.f) {
    g.R = dy; g.ldr = H; g.res_scale = alpha;
  }
  LAUNCH(FL_PROF_GEMM_NN, gemm_flops(T, H, F), gemm_bytes(T, H, F, E, E),
         gemm(dt, GEMM_NN, alpha > 0.f ? EPI_RES : EPI_STORE, with_part(g, plan), s));
  // w = LN2(h); h also feeds y directly (plain residual).  db_o = the column
  // sums of dh, formed in the same pass.
  if ((rc = ln_backward(st, dt, w.tmp, a.h, a.mean2, a.rstd2, p.ln2_g, alpha > 0.f ? nullptr : dy, w.dh, gr.ln2_g,
                        gr.ln2_b, train_w ? gr.b_o : nullptr, T, H, w, s)))
    return rc;
  // h = x + o W_o^T + b_o
  if (train_w) {
    g = GemmDesc();
    g.A = w.dh; g.B = a.o; g.C = gr.w_o; g.M = H; g.N = H; g.K = T; g.lda = H; g.ldb = H; g.ldc = H;
    LAUNCH(FL_PROF_GEMM_TN_ACC, gemm_flops(H, H, T), gemm_bytes(H, H, T, E, 8),
           gemm(dt, GEMM_TN, EPI_ACC_F32, with_part(g, plan), s));
  }
  g = GemmDesc();
  g.A = w.dh; g.B = p.w_o; g.C = w.tmp; g.M = T; g.N = H; g.K = H; g.lda = H; g.ldb = H; g.ldc = H;
  LAUNCH(FL_PROF_GEMM_NN, gemm_flops(T, H, H), gemm_bytes(T, H, H, E, E), gemm(dt, GEMM_NN, EPI_STORE, with_part(g, plan), s));
  // attention (dq, dk, dv with the inverse rotation applied)
  AttnDesc ad;
  ad.qkv = a.qkv; ad.ld_qkv = 3 * H; ad.o = a.o; ad.ld_o = H; ad.lse = a.lse;
  ad.cu_seqlens = plan.cu; ad.prefix_len = bi.prefix ? plan.prefix : nullptr;
  ad.num_seqs = bi.S; ad.max_seqlen = bi.maxL; ad.num_heads = st->d.num_heads; ad.head_dim = st->hd;
  ad.hidden = H; ad.total_tokens = T;
  ad.dout = w.tmp; ad.ld_dout = H; ad.delta = w.delta; ad.dqkv = w.dqkv; ad.ld_dqkv = 3 * H;
  // The attention kernels fuse the inverse rotation with the row's index
  // inside its sequence as the position; GLM 2-D positions differ from it
  // after the context, so in that mode both halves are rotated back below.
  ad.pos = plan.pos; ad.cos_t = plan.cos_t; ad.sin_t = plan.sin_t;
  ad.rotary_dim = st->d.rotary_2d ? 0 : st->d.rotary_dim;
  ad.pk = p.prefix_k; ad.pv = p.prefix_v; ad.num_prefix = st->d.num_prefix; ad.dprefix_part = w.dprefix;
  ad.ds = w.ds; ad.ds_off = w.ds_off;
  // b_qkv's column sums come from the attention kernels' own tiles (unless
  // the GLM 2-D rotation changes dq and dk after them)
  const bool fused_bqkv = train_w && w.ds && w.bias_part && !st->d.rotary_2d;
  if (fused_bqkv) {
    ad.bias_part = w.bias_part;
    ad.tile_base = w.tile_base;
  }
  const double pairs = bi.pairs + (double)st->d.num_prefix * T;
  LAUNCH(FL_PROF_ATTN_BWD, 8.0 * H * pairs, (double)T * H * E * 8, attn_bwd(dt, ad, s));
  if (st->d.rotary_2d)  // dq and dk rotated back: first half by p1, second by the block position
    LAUNCH(FL_PROF_ROPE, 0, 8.0 * T * st->d.num_heads * st->d.rotary_dim * E,
           rope_qk(dt, w.dqkv, 3 * H, plan.pos, plan.cos_t, plan.sin_t, T, H, st->hd, st->d.rotary_dim, s, -1.f,
                   plan.pos2));
  if (st->d.num_prefix) {
    // sum of the per-sequence prefix gradients, in sequence order
    const long n = (long)st->d.num_prefix * H;
    LAUNCH(FL_PROF_PREFIX_GRAD, 0, (2.0 * bi.S + 4.0) * n * 4,
           prefix_grad_reduce(w.dprefix, bi.S, n, gr.prefix_k, gr.prefix_v, s));
  }
  // qkv = u W_qkv^T + b_qkv
  if (train_w) {
    if (fused_bqkv)
      LAUNCH(FL_PROF_COLSUM, 0, 4.0 * w.bias_rows * 3 * H,
             colsum_finish(w.bias_part, w.bias_rows, 3 * H, gr.b_qkv, s));
    else if ((rc = colsum_into(st, dt, w.dqkv, 3 * H, T, 3 * H, gr.b_qkv, w, s)))
      return rc;
    g = GemmDesc();
    g.A = w.dqkv; g.B = a.u; g.C = gr.w_qkv; g.M = 3 * H; g.N = H; g.K = T; g.lda = 3 * H; g.ldb = H; g.ldc = H;
    LAUNCH(FL_PROF_GEMM_TN_ACC, gemm_flops(3 * H, H, T), gemm_bytes(3 * H, H, T, E, 8),
           gemm(dt, GEMM_TN, EPI_ACC_F32, with_part(g, plan), s));
  }
  g = GemmDesc();
  g.A = w.dqkv; g.B = p.w_qkv; g.C = w.tmp; g.M = T; g.N = H; g.K = 3 * H; g.lda = 3 * H; g.ldb = H; g.ldc = H;
  if (alpha > 0.f) {
    g.R = w.dh; g.ldr = H; g.res_scale = alpha;
  }
  LAUNCH(FL_PROF_GEMM_NN, gemm_flops(T, H, 3 * H), gemm_bytes(T, H, 3 * H, E, E),
         gemm(dt, GEMM_NN, alpha > 0.f ? EPI_RES : EPI_STORE, with_part(g, plan), s));
  // u = LN1(x); x also feeds h directly (plain residual)
  return ln_backward(st, dt, w.tmp, x, a.mean1, a.rstd1, p.ln1_g, alpha > 0.f ? nullptr : w.dh, dx, gr.ln1_g,
                     gr.ln1_b, dx_sum, T, H, w, s);
}

}  // namespace

namespace flglm {
int set_error(int code, const char* msg) { return fail(code, "%s", msg); }
}  // namespace flglm

// ---------------------------------------------------------------------------
// Allocation-free inference forward: the workspace is this file-scope device
// array (one per GPU, held until the process ends) instead of a caller
// buffer, and the batch plan travels in kernel arguments instead of through
// pinned host staging.
// ---------------------------------------------------------------------------
namespace {

constexpr size_t kScratchBytes = (size_t)FL_NOALLOC_SCRATCH_BYTES;
// Host code never uses this name as an address (it is a host-side stand-in
// there): it takes each device's address with hipGetSymbolAddress.
__device__ __align__(256) unsigned char scratch[kScratchBytes];

struct PlanArgs {
  int32_t num_seqs;
  int32_t cu[FL_NOALLOC_MAX_SEQS + 1];
  int32_t prefix[FL_NOALLOC_MAX_SEQS];
};
__global__ void plan_args_kernel(PlanArgs a, int32_t* cu, int32_t* prefix) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i <= a.num_seqs) cu[i] = a.cu[i];
  if (i < a.num_seqs) prefix[i] = a.prefix[i];
}

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch[kMaxDevices] = {};

// The scratch array's address on the current device, looked up once per
// device (with that device current) and kept.
int scratch_base(void** out) {
  int dev = -1;
  HIP_OK(hipGetDevice(&dev));
  if (dev < 0 || dev >= kMaxDevices) return fail(FL_ERR_HIP, "device %d outside [0, %d)", dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch[dev]) {
    void* ptr = nullptr;
    HIP_OK(hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)));
    if (!ptr) return fail(FL_ERR_HIP, "hipGetSymbolAddress gave no address for the scratch array");
    g_scratch[dev] = ptr;
  }
  *out = g_scratch[dev];
  return FL_OK;
}

// Launch timing records events; the allocation-free call turns it off for
// its own launches and restores it.
struct ProfOff {
  fl_stack* st;
  bool was;
  explicit ProfOff(fl_stack* s) : st(s), was(s->prof_mask) { st->prof_mask = 0; }
  ~ProfOff() { st->prof_mask = was; }
};

}  // namespace

// ===========================================================================
// C ABI
// ===========================================================================
extern "C" {

const char* fl_last_error(void) { return g_err.c_str(); }

int fl_stack_create(const fl_stack_desc* desc, fl_stack** out) {
  if (!out) return fail(FL_ERR_NULL, "out is NULL");
  *out = nullptr;
  int rc = validate_desc(desc);
  if (rc) return rc;
  // no exception may leave a C entry point: a failed allocation is an error code
  fl_stack* st = new (std::nothrow) fl_stack();
  if (!st) return fail(FL_ERR_NOMEM, "out of host memory for the stack handle");
  st->d = *desc;
  st->E = desc->dtype == FL_BF16 ? 2 : 4;
  st->hd = desc->hidden / desc->num_heads;
  *out = st;
  return FL_OK;
}

int fl_stack_destroy(fl_stack* st) {
  if (!st) return FL_OK;
  int rc = FL_OK;
  for (auto& r : st->recs) {
    st->pool.push_back(r.a);
    st->pool.push_back(r.b);
  }
  for (hipEvent_t e : st->pool)
    if (hipEventDestroy(e) != hipSuccess) rc = FL_ERR_HIP;
  for (int k = 0; k < fl_stack::kRing; ++k) {
    if (st->ev_used[k] && hipEventSynchronize(st->ev[k]) != hipSuccess) rc = FL_ERR_HIP;
    if (st->stage[k] && hipHostFree(st->stage[k]) != hipSuccess) rc = FL_ERR_HIP;
    if (st->ev_made[k] && hipEventDestroy(st->ev[k]) != hipSuccess) rc = FL_ERR_HIP;
  }
  delete st;
  if (rc) return fail(rc, "HIP error while releasing the handle");
  return FL_OK;
}

int fl_stack_profile_classes(fl_stack* st, uint32_t class_mask) {
  if (!st) return fail(FL_ERR_NULL, "stack is NULL");
  class_mask &= (1u << FL_PROF_NUM_CLASSES) - 1u;
  if (class_mask) {
    for (auto& r : st->recs) {
      st->pool.push_back(r.a);
      st->pool.push_back(r.b);
    }
    st->recs.clear();
  }
  st->prof_mask = class_mask;
  return FL_OK;
}

int fl_stack_profile(fl_stack* st, int enable) {
  return fl_stack_profile_classes(st, enable ? (1u << FL_PROF_NUM_CLASSES) - 1u : 0u);
}

int fl_stack_profile_read(fl_stack* st, int cls, int64_t* launches, double* ms, double* flops, double* bytes) {
  if (!st || !launches || !ms || !flops || !bytes) return fail(FL_ERR_NULL, "NULL argument");
  if (cls < 0 || cls >= FL_PROF_NUM_CLASSES) return fail(FL_ERR_ARG, "profile class %d out of range", cls);
  *launches = 0;
  *ms = *flops = *bytes = 0.0;
  for (auto& r : st->recs) {
    if (r.cls != cls) continue;
    HIP_OK(hipEventSynchronize(r.b));
    float t = 0.f;
    HIP_OK(hipEventElapsedTime(&t, r.a, r.b));
    *launches += 1;
    *ms += t;
    *flops += r.flops;
    *bytes += r.bytes;
  }
  return FL_OK;
}

const char* fl_profile_class_name(int cls) {
  return (cls >= 0 && cls < FL_PROF_NUM_CLASSES) ? kProfNames[cls] : "";
}

int fl_stack_saved_bytes(const fl_stack* st, const fl_batch_desc* b, int recompute, size_t* bytes) {
  if (!st || !bytes) return fail(FL_ERR_NULL, "stack / bytes is NULL");
  BatchInfo bi;
  int rc = validate_batch(b, &bi);
  if (rc) return rc;
  *bytes = saved_bytes(st, bi, recompute != 0);
  return FL_OK;
}

int fl_stack_workspace_bytes(const fl_stack* st, const fl_batch_desc* b, int recompute, size_t* bytes) {
  (void)recompute;
  if (!st || !bytes) return fail(FL_ERR_NULL, "stack / bytes is NULL");
  BatchInfo bi;
  int rc = validate_batch(b, &bi);
  if (rc) return rc;
  *bytes = work_bytes(st, bi);
  return FL_OK;
}

int fl_client_token_range(const fl_batch_desc* b, int32_t client, int64_t* begin, int64_t* end) {
  if (!begin || !end) return fail(FL_ERR_NULL, "begin / end is NULL");
  BatchInfo bi;
  int rc = validate_batch(b, &bi);
  if (rc) return rc;
  if (client < 0 || client >= bi.C) return fail(FL_ERR_ARG, "client %d outside [0, %d)", client, bi.C);
  *begin = b->cu_seqlens[b->client_seq_ptr[client]];
  *end = b->cu_seqlens[b->client_seq_ptr[client + 1]];
  return FL_OK;
}

int fl_server_stack_forward(fl_stack* st, const fl_batch_desc* b, const fl_layer_params* layers, const void* x,
                            void* y, void* saved, int recompute, void* ws, size_t ws_bytes, void* stream) {
  if (!st) return fail(FL_ERR_NULL, "stack is NULL");
  BatchInfo bi;
  int rc = validate_batch(b, &bi);
  if (rc) return rc;
  if ((rc = check_params(st, layers))) return rc;
  if (!x || !y || !ws) return fail(FL_ERR_NULL, "x / y / workspace is NULL");
  if (!aligned16(x) || !aligned16(y) || !aligned16(ws) || (saved && !aligned16(saved)))
    return fail(FL_ERR_ALIGN, "x / y / saved / workspace must be 16-byte aligned");
  const size_t need_ws = work_bytes(st, bi);
  if (ws_bytes < need_ws) return fail(FL_ERR_WORKSPACE, "workspace %zu bytes < required %zu", ws_bytes, need_ws);
  const size_t act = (size_t)st->E * bi.T * st->d.hidden;
  const size_t nsaved = saved ? saved_bytes(st, bi, recompute != 0) : 0;
  if (overlap(x, act, y, act)) return fail(FL_ERR_ALIAS, "y overlaps x");
  if (overlap(ws, ws_bytes, x, act) || overlap(ws, ws_bytes, y, act) || overlap(ws, ws_bytes, saved, nsaved))
    return fail(FL_ERR_ALIAS, "workspace overlaps x / y / saved");
  if (overlap(saved, nsaved, x, act) || overlap(saved, nsaved, y, act))
    return fail(FL_ERR_ALIAS, "saved overlaps x / y");

  hipStream_t s = (hipStream_t)stream;
  Carver cw(ws);
  Work w;
  carve_work(cw, st, bi, &w);
  Saved sv;
  if (saved) {
    Carver cs(saved);
    carve_saved(cs, st, bi.T, recompute != 0, &sv);
  }
  if ((rc = upload_plan(st, b, bi, w.plan, s))) return rc;
  const int N = st->d.num_layers;
  const void* cur = x;
  for (int l = 0; l < N; ++l) {
    const bool keep = saved && !recompute;  // intermediates kept for the backward
    const Acts& a = keep ? sv.acts[l] : w.acts;
    void* out = (l == N - 1) ? y : (saved ? sv.xin[l + 1] : w.ping[l & 1]);
    if ((rc = block_forward(st, bi, w.plan, layers[l], cur, a, out, s, keep))) return rc;
    cur = out;
  }
  return FL_OK;
}

int fl_server_stack_forward_noalloc(fl_stack* st, const fl_batch_desc* b, const fl_layer_params* layers,
                                    const void* x, void* y, void* stream) {
  if (!st) return fail(FL_ERR_NULL, "stack is NULL");
  BatchInfo bi;
  int rc = validate_batch(b, &bi);
  if (rc) return rc;
  if (bi.S > FL_NOALLOC_MAX_SEQS)
    return fail(FL_ERR_ARG, "%d sequences: the allocation-free forward takes at most %d", bi.S, FL_NOALLOC_MAX_SEQS);
  if ((rc = check_params(st, layers))) return rc;
  if (!x || !y) return fail(FL_ERR_NULL, "x / y is NULL");
  if (!aligned16(x) || !aligned16(y)) return fail(FL_ERR_ALIGN, "x / y must be 16-byte aligned");
  const size_t need = fwd_work_bytes(st, bi);
  if (need > kScratchBytes)
    return fail(FL_ERR_WORKSPACE, "batch of %d tokens needs %zu bytes of scratch; the static scratch holds %zu", bi.T,
                need, kScratchBytes);
  const size_t act = (size_t)st->E * bi.T * st->d.hidden;
  if (overlap(x, act, y, act)) return fail(FL_ERR_ALIAS, "y overlaps x");
  void* base = nullptr;
  if ((rc = scratch_base(&base))) return rc;
  if (overlap(base, kScratchBytes, x, act) || overlap(base, kScratchBytes, y, act))
    return fail(FL_ERR_ALIAS, "x / y overlap the library's scratch array");

  hipStream_t s = (hipStream_t)stream;
  Carver cw(base);
  Work w;
  carve_fwd_work(cw, st, bi, &w);
  PlanArgs pa;
  pa.num_seqs = bi.S;
  std::memcpy(pa.cu, b->cu_seqlens, sizeof(int32_t) * (bi.S + 1));
  if (bi.prefix) std::memcpy(pa.prefix, b->prefix_len, sizeof(int32_t) * bi.S);
  else std::memset(pa.prefix, 0, sizeof(int32_t) * bi.S);
  ProfOff off(st);
  hipLaunchKernelGGL(plan_args_kernel, dim3((bi.S + 1 + 255) / 256), dim3(256), 0, s, pa, w.plan.cu, w.plan.prefix);
  HIP_OK(hipGetLastError());
  if ((rc = plan_kernels(st, bi, w.plan, s))) return rc;
  const int N = st->d.num_layers;
  const void* cur = x;
  for (int l = 0; l < N; ++l) {
    void* out = (l == N - 1) ? y : w.ping[l & 1];
    if ((rc = block_forward(st, bi, w.plan, layers[l], cur, w.acts, out, s, false))) return rc;
    cur = out;
  }
  return FL_OK;
}

int fl_server_stack_backward(fl_stack* st, const fl_batch_desc* b, const fl_layer_params* layers,
                             const fl_layer_grads* grads, const void* x, const void* saved, const void* dy, void* dx,
                             int recompute, void* ws, size_t ws_bytes, void* stream) {
  if (!st) return fail(FL_ERR_NULL, "stack is NULL");
  BatchInfo bi;
  int rc = validate_batch(b, &bi);
  if (rc) return rc;
  if ((rc = check_params(st, layers))) return rc;
  if ((rc = check_grads(st, grads))) return rc;
  if (!x || !saved || !dy || !dx || !ws) return fail(FL_ERR_NULL, "x / saved / dy / dx / workspace is NULL");
  if (!aligned16(x) || !aligned16(saved) || !aligned16(dy) || !aligned16(dx) || !aligned16(ws))
    return fail(FL_ERR_ALIGN, "x / saved / dy / dx / workspace must be 16-byte aligned");
  const size_t need_ws = work_bytes(st, bi);
  if (ws_bytes < need_ws) return fail(FL_ERR_WORKSPACE, "workspace %zu bytes < required %zu", ws_bytes, need_ws);
  const size_t act = (size_t)st->E * bi.T * st->d.hidden;
  const size_t nsaved = saved_bytes(st, bi, recompute != 0);
  if (overlap(dx, act, dy, act) || overlap(dx, act, x, act) || overlap(dx, act, saved, nsaved))
    return fail(FL_ERR_ALIAS, "dx overlaps dy / x / saved");
  if (overlap(ws, ws_bytes, x, act) || overlap(ws, ws_bytes, dy, act) || overlap(ws, ws_bytes, dx, act) ||
      overlap(ws, ws_bytes, saved, nsaved))
    return fail(FL_ERR_ALIAS, "workspace overlaps x / saved / dy / dx");

  hipStream_t s = (hipStream_t)stream;
  Carver cw(ws);
  Work w;
  carve_work(cw, st, bi, &w);
  Saved sv;
  Carver cs(const_cast<void*>(saved));
  carve_saved(cs, st, bi.T, recompute != 0, &sv);
  if ((rc = upload_plan(st, b, bi, w.plan, s))) return rc;
  const int N = st->d.num_layers;
  const void* gcur = dy;
  for (int l = N - 1; l >= 0; --l) {
    const void* xin = (l == 0) ? x : sv.xin[l];
    const Acts* a = &sv.acts[l];
    if (recompute) {
      if ((rc = block_forward(st, bi, w.plan, layers[l], xin, w.acts, nullptr, s))) return rc;
      a = &w.acts;
    }
    void* gout = (l == 0) ? dx : w.ping[(N - 1 - l) & 1];
    // block l's dx is block l - 1's dy: its column sums (block l - 1's db_2)
    // come out of block l's last LayerNorm backward
    float* below_b2 = l > 0 ? grads[l - 1].b_2 : nullptr;
    const bool b2_done = l < N - 1 && grads[l].b_2 != nullptr;
    if ((rc = block_backward(st, bi, w.plan, w, layers[l], grads[l], xin, *a, gcur, gout, s, below_b2, b2_done)))
      return rc;
    gcur = gout;
  }
  return FL_OK;
}

static int pack_impl(fl_stack* st, const fl_batch_desc* b, const void* const* cbufs, void* packed, void* ws,
                     size_t ws_bytes, void* stream, bool unpack) {
  if (!st) return fail(FL_ERR_NULL, "stack is NULL");
  BatchInfo bi;
  int rc = validate_batch(b, &bi);
  if (rc) return rc;
  if (!cbufs || !packed || !ws) return fail(FL_ERR_NULL, "client buffers / packed / workspace is NULL");
  if (!aligned16(packed) || !aligned16(ws)) return fail(FL_ERR_ALIGN, "packed / workspace must be 16-byte aligned");
  for (int c = 0; c < bi.C; ++c) {
    if (!cbufs[c]) return fail(FL_ERR_NULL, "client buffer %d is NULL", c);
    if (!aligned16(cbufs[c])) return fail(FL_ERR_ALIGN, "client buffer %d is not 16-byte aligned", c);
  }
  const size_t need_ws = work_bytes(st, bi);
  if (ws_bytes < need_ws) return fail(FL_ERR_WORKSPACE, "workspace %zu bytes < required %zu", ws_bytes, need_ws);
  hipStream_t s = (hipStream_t)stream;
  Carver cw(ws);
  Work w;
  carve_work(cw, st, bi, &w);
  if ((rc = upload_plan(st, b, bi, w.plan, s))) return rc;
  for (int c = 0; c < bi.C; ++c) {
    const int s0 = b->client_seq_ptr[c], s1 = b->client_seq_ptr[c + 1];
    int Lmax = 0;
    for (int q = s0; q < s1; ++q) Lmax = std::max(Lmax, b->cu_seqlens[q + 1] - b->cu_seqlens[q]);
    HIP_OK(pack_client((DType)st->d.dtype, cbufs[c], packed, w.plan.cu, s0, s1 - s0, Lmax, st->d.hidden, unpack, s));
  }
  return FL_OK;
}

int fl_pack_clients(fl_stack* st, const fl_batch_desc* b, const void* const* cbufs, void* packed, void* ws,
                    size_t ws_bytes, void* stream) {
  return pack_impl(st, b, cbufs, packed, ws, ws_bytes, stream, false);
}

int fl_unpack_clients(fl_stack* st, const fl_batch_desc* b, const void* packed, void* const* cbufs, void* ws,
                      size_t ws_bytes, void* stream) {
  return pack_impl(st, b, (const void* const*)cbufs, const_cast<void*>(packed), ws, ws_bytes, stream, true);
}

}  // extern "C"
