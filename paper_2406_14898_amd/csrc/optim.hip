// Server update after the backward pass, and its C ABI entry points.
//
//  * Adam (Kingma & Ba, Algorithm 1), the optimizer the paper trains with
//    (Section 4.1.4: learning rate 2e-2, no warmup, no weight decay), over a
//    flat fp32 master copy with its fp32 gradient and moments; optionally
//    refreshes the bf16 compute copy and clears the gradient for the next
//    accumulation in the same pass.
//  * Replica averaging of the server-hierarchical strategy (Section 3.3: one
//    server-side model per client, parameters averaged at the end of each
//    training period): every replica receives the elementwise mean.
//
// Both are pure streams over HBM: 16-byte vector accesses, four elements per
// lane, non-temporal loads and stores (nothing is re-read, so nothing is worth
// keeping in the caches; measured +8 % over cached accesses for Adam's nine
// streams), all arithmetic in fp32.
#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>

#include "../../include/flglm.h"
#include "common.h"

namespace flglm {
int set_error(int code, const char* msg);
}

using namespace flglm;

namespace {

__device__ __forceinline__ f32x4 ld_nt(const float* p) {
  return __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(p));
}
__device__ __forceinline__ void st_nt(float* p, f32x4 v) { __builtin_nontemporal_store(v, reinterpret_cast<f32x4*>(p)); }
__device__ __forceinline__ void st_nt(bf16* p, const float (&v)[4]) {
  const bf16x4 b = {from_f32<bf16>(v[0]), from_f32<bf16>(v[1]), from_f32<bf16>(v[2]), from_f32<bf16>(v[3])};
  __builtin_nontemporal_store(__builtin_bit_cast(u32x2, b), reinterpret_cast<u32x2*>(p));
}

constexpr int kThreads = 256;
constexpr int kUnroll = 1;                       // float4 groups per thread (1 measured best)
constexpr long kPerBlock = 4L * kThreads * kUnroll;
constexpr int kMaxReplicas = 32;

struct AdamArgs {
  float* p;
  float* g;
  float* m;
  float* v;
  bf16* p16;  // nullable
  long n;
  float lr, beta1, beta2, one_m_beta1, one_m_beta2, bc1, bc2, eps;
  int zero_grad;
};

// One element of Algorithm 1 in its order: moments, bias corrections, step.
__device__ __forceinline__ void adam_elem(const AdamArgs& a, float& p, float g, float& m, float& v) {
  m = a.beta1 * m + a.one_m_beta1 * g;
  v = a.beta2 * v + a.one_m_beta2 * (g * g);
  const float m_hat = m / a.bc1;
  const float v_hat = v / a.bc2;
  p = p - a.lr * m_hat / (sqrtf(v_hat) + a.eps);
}

__global__ void __launch_bounds__(kThreads) adam_kernel(AdamArgs a) {
  const long base = (long)blockIdx.x * kPerBlock + (long)threadIdx.x * 4;
  long e[kUnroll];
  bool full[kUnroll];
  f32x4 P[kUnroll], G[kUnroll], M[kUnroll], V[kUnroll];
#pragma unroll
  for (int u = 0; u < kUnroll; ++u) {
    e[u] = base + (long)u * 4 * kThreads;
    full[u] = e[u] + 4 <= a.n;
    if (full[u]) {
      P[u] = ld_nt(a.p + e[u]);
      G[u] = ld_nt(a.g + e[u]);
      M[u] = ld_nt(a.m + e[u]);
      V[u] = ld_nt(a.v + e[u]);
    }
  }
#pragma unroll
  for (int u = 0; u < kUnroll; ++u) {
    if (full[u]) {
      float p[4], m[4], v[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        p[i] = P[u][i];
        m[i] = M[u][i];
        v[i] = V[u][i];
        adam_elem(a, p[i], G[u][i], m[i], v[i]);
      }
      st_nt(a.p + e[u], f32x4{p[0], p[1], p[2], p[3]});
      st_nt(a.m + e[u], f32x4{m[0], m[1], m[2], m[3]});
      st_nt(a.v + e[u], f32x4{v[0], v[1], v[2], v[3]});
      if (a.p16) st_nt(a.p16 + e[u], p);
      if (a.zero_grad) st_nt(a.g + e[u], f32x4{0.f, 0.f, 0.f, 0.f});
    } else if (e[u] < a.n) {
      // ragged tail: fewer than four elements left, element by element
      for (long j = e[u]; j < a.n; ++j) {
        float p = a.p[j], m = a.m[j], v = a.v[j];
        adam_elem(a, p, a.g[j], m, v);
        a.p[j] = p;
        a.m[j] = m;
        a.v[j] = v;
        if (a.p16) a.p16[j] = from_f32<bf16>(p);
        if (a.zero_grad) a.g[j] = 0.f;
      }
    }
  }
}

struct AvgArgs {
  float* rep[kMaxReplicas];
  bf16* rep16[kMaxReplicas];  // all NULL or all set
  int num;
  long n;
};

__global__ void __launch_bounds__(kThreads) average_kernel(AvgArgs a) {
  const long base = (long)blockIdx.x * kPerBlock + (long)threadIdx.x * 4;
  const float num_f = (float)a.num;
#pragma unroll
  for (int u = 0; u < kUnroll; ++u) {
    const long e = base + (long)u * 4 * kThreads;
    if (e + 4 <= a.n) {
      float s[4] = {0.f, 0.f, 0.f, 0.f};
      for (int r = 0; r < a.num; ++r) {  // replica order is the summation order
        const f32x4 x = ld_nt(a.rep[r] + e);
#pragma unroll
        for (int i = 0; i < 4; ++i) s[i] += x[i];
      }
      float mean[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) mean[i] = s[i] / num_f;
      for (int r = 0; r < a.num; ++r) {
        st_nt(a.rep[r] + e, f32x4{mean[0], mean[1], mean[2], mean[3]});
        if (a.rep16[0]) st_nt(a.rep16[r] + e, mean);
      }
    } else if (e < a.n) {
      for (long j = e; j < a.n; ++j) {
        float s = 0.f;
        for (int r = 0; r < a.num; ++r) s += a.rep[r][j];
        const float mean = s / num_f;
        for (int r = 0; r < a.num; ++r) {
          a.rep[r][j] = mean;
          if (a.rep16[0]) a.rep16[r][j] = from_f32<bf16>(mean);
        }
      }
    }
  }
}

bool al16(const void* p) { return ((uintptr_t)p & 15) == 0; }

bool overlap(const void* a, size_t na, const void* b, size_t nb) {
  const uintptr_t x = (uintptr_t)a, y = (uintptr_t)b;
  return x < y + nb && y < x + na;
}

int launch_status() {
  const hipError_t e = hipGetLastError();
  return e == hipSuccess ? FL_OK : set_error(FL_ERR_HIP, hipGetErrorString(e));
}

unsigned grid_for(long n) { return (unsigned)((n + kPerBlock - 1) / kPerBlock); }

}  // namespace

extern "C" {

int fl_adam_step(float* param, float* grad, float* exp_avg, float* exp_avg_sq, void* param_bf16, int64_t n,
                 int64_t step, double lr, double beta1, double beta2, double eps, int zero_grad, void* stream) {
  if (!param || !grad || !exp_avg || !exp_avg_sq) return set_error(FL_ERR_NULL, "param / grad / moments NULL");
  if (!al16(param) || !al16(grad) || !al16(exp_avg) || !al16(exp_avg_sq) || !al16(param_bf16))
    return set_error(FL_ERR_ALIGN, "Adam buffers must be 16-byte aligned");
  if (n < 0 || n > (int64_t(1) << 40)) return set_error(FL_ERR_ARG, "bad element count");
  if (step < 1) return set_error(FL_ERR_ARG, "Adam time steps start at 1");
  if (!(std::isfinite(lr) && lr >= 0.0) || !(beta1 >= 0.0 && beta1 < 1.0) || !(beta2 >= 0.0 && beta2 < 1.0) ||
      !(std::isfinite(eps) && eps >= 0.0))
    return set_error(FL_ERR_ARG, "bad Adam hyper-parameters");
  if (zero_grad != 0 && zero_grad != 1) return set_error(FL_ERR_ARG, "zero_grad must be 0 or 1");
  const size_t b4 = (size_t)n * 4;
  const void* bufs[5] = {param, grad, exp_avg, exp_avg_sq, param_bf16};
  const size_t sizes[5] = {b4, b4, b4, b4, (size_t)n * 2};
  for (int i = 0; i < 5; ++i)
    for (int j = i + 1; j < 5; ++j)
      if (bufs[i] && bufs[j] && overlap(bufs[i], sizes[i], bufs[j], sizes[j]))
        return set_error(FL_ERR_ALIAS, "Adam buffers overlap");
  // 1 - beta and the bias corrections 1 - beta^t in double, each rounded once
  // to fp32 (beta close to 1 would lose digits if subtracted in fp32)
  const double bc1 = 1.0 - std::pow(beta1, (double)step);
  const double bc2 = 1.0 - std::pow(beta2, (double)step);
  if (!(bc1 > 0.0) || !(bc2 > 0.0)) return set_error(FL_ERR_ARG, "bias correction 1 - beta^step rounds to zero");
  if (n == 0) return FL_OK;
  AdamArgs a;
  a.p = param; a.g = grad; a.m = exp_avg; a.v = exp_avg_sq; a.p16 = (bf16*)param_bf16; a.n = n;
  a.lr = (float)lr; a.beta1 = (float)beta1; a.beta2 = (float)beta2;
  a.one_m_beta1 = (float)(1.0 - beta1); a.one_m_beta2 = (float)(1.0 - beta2);
  a.bc1 = (float)bc1; a.bc2 = (float)bc2; a.eps = (float)eps; a.zero_grad = zero_grad;
  hipLaunchKernelGGL(adam_kernel, dim3(grid_for(n)), dim3(kThreads), 0, (hipStream_t)stream, a);
  return launch_status();
}

int fl_average_replicas(int32_t num_replicas, float* const* params, void* const* params_bf16, int64_t n,
                        void* stream) {
  if (num_replicas < 1 || num_replicas > kMaxReplicas) return set_error(FL_ERR_ARG, "1 <= num_replicas <= 32");
  if (!params) return set_error(FL_ERR_NULL, "params NULL");
  if (n < 0 || n > (int64_t(1) << 40)) return set_error(FL_ERR_ARG, "bad element count");
  AvgArgs a = {};
  a.num = num_replicas;
  a.n = n;
  for (int r = 0; r < num_replicas; ++r) {
    if (!params[r] || (params_bf16 && !params_bf16[r])) return set_error(FL_ERR_NULL, "a replica pointer is NULL");
    if (!al16(params[r]) || (params_bf16 && !al16(params_bf16[r])))
      return set_error(FL_ERR_ALIGN, "replica buffers must be 16-byte aligned");
    a.rep[r] = params[r];
    a.rep16[r] = params_bf16 ? (bf16*)params_bf16[r] : nullptr;
  }
  // every buffer is written: no two may overlap
  const int nb = params_bf16 ? 2 * num_replicas : num_replicas;
  for (int i = 0; i < nb; ++i)
    for (int j = i + 1; j < nb; ++j) {
      const void* x = i < num_replicas ? (const void*)a.rep[i] : (const void*)a.rep16[i - num_replicas];
      const void* y = j < num_replicas ? (const void*)a.rep[j] : (const void*)a.rep16[j - num_replicas];
      const size_t nx = (size_t)n * (i < num_replicas ? 4 : 2), ny = (size_t)n * (j < num_replicas ? 4 : 2);
      if (overlap(x, nx, y, ny)) return set_error(FL_ERR_ALIAS, "replica buffers overlap");
    }
  if (n == 0) return FL_OK;
  hipLaunchKernelGGL(average_kernel, dim3(grid_for(n)), dim3(kThreads), 0, (hipStream_t)stream, a);
  return launch_status();
}

}  // extern "C"
