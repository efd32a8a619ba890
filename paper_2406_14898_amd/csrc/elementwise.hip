// Memory-bound kernels of the block: LayerNorm forward/backward, rotary
// position encoding, deterministic column sums (bias and LayerNorm parameter
// gradients), packed-batch bookkeeping and client packing.  All of them move
// 16-byte vectors along the contiguous hidden dimension.
#include "common.h"
#include "kernels.h"

namespace flglm {

// ---------------------------------------------------------------------------
// Positions and rotary table
// ---------------------------------------------------------------------------
__global__ void seq_positions_kernel(const int32_t* cu, int32_t* pos) {
  const int s = blockIdx.x;
  const int r0 = cu[s], r1 = cu[s + 1];
  for (int r = r0 + (int)threadIdx.x; r < r1; r += blockDim.x) pos[r] = r - r0;
}

hipError_t seq_positions(const int32_t* cu, int S, int32_t* pos, hipStream_t st) {
  if (S <= 0) return hipSuccess;
  hipLaunchKernelGGL(seq_positions_kernel, dim3(S), dim3(256), 0, st, cu, pos);
  return hipGetLastError();
}

// GLM 2-D positions: with a context of P tokens (ctx[s], or the whole
// sequence), p1 = t inside the context and the [gMASK] position max(P-1, 0)
// after it; p2 = 0 inside the context and t - P + 1 after it.
__global__ void seq_positions_2d_kernel(const int32_t* cu, const int32_t* ctx, int32_t* p1, int32_t* p2) {
  const int s = blockIdx.x;
  const int r0 = cu[s], r1 = cu[s + 1];
  const int P = ctx ? ctx[s] : r1 - r0;
  const int m = P > 0 ? P - 1 : 0;
  for (int r = r0 + (int)threadIdx.x; r < r1; r += blockDim.x) {
    const int t = r - r0;
    p1[r] = t < P ? t : m;
    p2[r] = t < P ? 0 : t - P + 1;
  }
}

hipError_t seq_positions_2d(const int32_t* cu, const int32_t* ctx, int S, int32_t* p1, int32_t* p2, hipStream_t st) {
  if (S <= 0) return hipSuccess;
  hipLaunchKernelGGL(seq_positions_2d_kernel, dim3(S), dim3(256), 0, st, cu, ctx, p1, p2);
  return hipGetLastError();
}

__global__ void rope_table_kernel(float* ct, float* stbl, int max_pos, int r, double base) {
  const int half = r / 2;
  const long idx = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= (long)max_pos * half) return;
  const int p = (int)(idx / half), i = (int)(idx % half);
  const double theta = pow(base, -2.0 * (double)i / (double)r);
  const double ang = (double)p * theta;
  ct[idx] = (float)cos(ang);
  stbl[idx] = (float)sin(ang);
}

hipError_t rope_table(float* ct, float* stbl, int max_pos, int r, float base, hipStream_t st) {
  const long n = (long)max_pos * (r / 2);
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(rope_table_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, st, ct, stbl, max_pos,
                     r, (double)base);
  return hipGetLastError();
}

// One thread rotates 8 pairs (i, i + r/2), i..i+7, of one head of q or k
// (16-byte loads for bf16; r / 2 is a multiple of 8).
template <typename T>
// pos2 (GLM 2-D positions): the same thread also rotates the matching pairs
// of dims [r, 2r) by pos2, so both halves take one pass over q and k.
__global__ void rope_qk_kernel(T* qkv, long ld, const int32_t* pos, const int32_t* pos2, const float* ct,
                               const float* stbl, int T_, int H, int d, int r, float sign) {
  const int half = r / 2, groups = half / 8;
  const int nh = H / d;
  const long idx = (long)blockIdx.x * blockDim.x + threadIdx.x;
  const long per_row = 2L * nh * groups;
  if (idx >= (long)T_ * per_row) return;
  const int t = (int)(idx / per_row);
  int rem = (int)(idx % per_row);
  const int part = rem / (nh * groups);
  rem %= nh * groups;
  const int h = rem / groups, i = (rem % groups) * 8;
  T* base = qkv + (long)t * ld + part * H + h * d;
  auto rotate = [&](int off, int p) {
    Vec8<T> a, b;
    a.load(base + off + i);
    b.load(base + off + half + i);
    Vec8<float> c, sn;
    c.load(ct + (long)p * half + i);
    sn.load(stbl + (long)p * half + i);
    float ya[8], yb[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float x1 = a.get(e), x2 = b.get(e), se = sign * sn.get(e);
      ya[e] = x1 * c.get(e) - x2 * se;
      yb[e] = x2 * c.get(e) + x1 * se;
    }
    a.set(ya);
    b.set(yb);
    a.store(base + off + i);
    b.store(base + off + half + i);
  };
  rotate(0, pos[t]);
  if (pos2) rotate(r, pos2[t]);
}

hipError_t rope_qk(DType dt, void* qkv, long ld, const int32_t* pos, const float* ct, const float* stbl, int T_,
                   int H, int d, int r, hipStream_t st, float sign, const int32_t* pos2) {
  const long n = (long)T_ * 2 * (H / d) * (r / 16);
  if (n <= 0) return hipSuccess;
  if (r % 16 != 0) return hipErrorInvalidValue;
  dim3 g((unsigned)((n + 255) / 256));
  if (dt == DT_BF16)
    hipLaunchKernelGGL(rope_qk_kernel<bf16>, g, dim3(256), 0, st, (bf16*)qkv, ld, pos, pos2, ct, stbl, T_, H, d, r,
                       sign);
  else
    hipLaunchKernelGGL(rope_qk_kernel<float>, g, dim3(256), 0, st, (float*)qkv, ld, pos, pos2, ct, stbl, T_, H, d,
                       r, sign);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// LayerNorm: one wave per row, the row held in registers in its storage
// type (MAXC 8-element chunks per lane, H <= 512 * MAXC) and converted on
// each of the three passes: half the registers of an fp32 copy for bf16
// rows, so twice as many rows are in flight per CU.
// ---------------------------------------------------------------------------
template <typename T, int MAXC>
__global__ void __launch_bounds__(256) ln_fwd_kernel(const T* x, const T* g, const T* b, T* y, float* mean,
                                                     float* rstd, int T_, int H, float eps) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= T_) return;
  const int nch = H / 8;
  const T* xr = x + (long)row * H;
  Vec8<T> v[MAXC];
#pragma unroll
  for (int c = 0; c < MAXC; ++c) {
    const int idx = lane + 64 * c;
    if (idx < nch) v[c].load(xr + idx * 8);
    else v[c].zero();
  }
  float s = 0.f;
#pragma unroll
  for (int c = 0; c < MAXC; ++c)
#pragma unroll
    for (int e = 0; e < 8; ++e) s += v[c].get(e);
  const float mu = wave_sum(s) / (float)H;
#pragma unroll
  for (int c = 0; c < MAXC; ++c) v[c].settle();
  float ss = 0.f;
#pragma unroll
  for (int c = 0; c < MAXC; ++c) {
    if (lane + 64 * c < nch) {
#pragma unroll
      for (int e = 0; e < 8; ++e) { const float dlt = v[c].get(e) - mu; ss += dlt * dlt; }
    }
  }
  const float rs = 1.0f / sqrtf(wave_sum(ss) / (float)H + eps);
#pragma unroll
  for (int c = 0; c < MAXC; ++c) v[c].settle();
  T* yr = y + (long)row * H;
#pragma unroll
  for (int c = 0; c < MAXC; ++c) {
    const int idx = lane + 64 * c;
    if (idx < nch) {
      Vec8<T> gg, bb, o;
      gg.load(g + idx * 8);
      bb.load(b + idx * 8);
      float out[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) out[e] = (v[c].get(e) - mu) * rs * gg.get(e) + bb.get(e);
      o.set(out);
      o.store(yr + idx * 8);
    }
  }
  if (lane == 0) { mean[row] = mu; rstd[row] = rs; }
}

template <typename T, int MAXC>
__global__ void __launch_bounds__(256) ln_bwd_dx_kernel(const T* dy, const T* x, const float* mean,
                                                        const float* rstd, const T* g, const T* dres, T* dx, int T_,
                                                        int H) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= T_) return;
  const int nch = H / 8;
  const float mu = mean[row], rs = rstd[row];
  const long off = (long)row * H;
  float dxh[MAXC][8], xh[MAXC][8];
  float s1 = 0.f, s2 = 0.f;
#pragma unroll
  for (int c = 0; c < MAXC; ++c) {
    const int idx = lane + 64 * c;
    if (idx < nch) {
      Vec8<T> a, xx, gg;
      a.load(dy + off + idx * 8);
      xx.load(x + off + idx * 8);
      gg.load(g + idx * 8);
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        xh[c][e] = (xx.get(e) - mu) * rs;
        dxh[c][e] = a.get(e) * gg.get(e);
        s1 += dxh[c][e];
        s2 += dxh[c][e] * xh[c][e];
      }
    }
  }
  const float m1 = wave_sum(s1) / (float)H;
  const float m2 = wave_sum(s2) / (float)H;
#pragma unroll
  for (int c = 0; c < MAXC; ++c) {
    const int idx = lane + 64 * c;
    if (idx < nch) {
      Vec8<T> r, o;
      if (dres)
        r.load(dres + off + idx * 8);
      else
        r.zero();
      float out[8];
#pragma unroll
      for (int e = 0; e < 8; ++e) out[e] = r.get(e) + rs * (dxh[c][e] - m1 - xh[c][e] * m2);
      o.set(out);
      o.store(dx + off + idx * 8);
    }
  }
}

template <typename T>
static hipError_t ln_fwd_t(const void* x, const void* g, const void* b, void* y, float* mean, float* rstd, int T_,
                           int H, float eps, hipStream_t st) {
  dim3 grid((T_ + 3) / 4), blk(256);
  const int nch = H / 8;
  if (nch <= 64)
    hipLaunchKernelGGL((ln_fwd_kernel<T, 1>), grid, blk, 0, st, (const T*)x, (const T*)g, (const T*)b, (T*)y, mean,
                       rstd, T_, H, eps);
  else if (nch <= 256)
    hipLaunchKernelGGL((ln_fwd_kernel<T, 4>), grid, blk, 0, st, (const T*)x, (const T*)g, (const T*)b, (T*)y, mean,
                       rstd, T_, H, eps);
  else if (nch <= 512)
    hipLaunchKernelGGL((ln_fwd_kernel<T, 8>), grid, blk, 0, st, (const T*)x, (const T*)g, (const T*)b, (T*)y, mean,
                       rstd, T_, H, eps);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

template <typename T>
static hipError_t ln_bwd_t(const void* dy, const void* x, const float* mean, const float* rstd, const void* g,
                           const void* dres, void* dx, int T_, int H, hipStream_t st) {
  dim3 grid((T_ + 3) / 4), blk(256);
  const int nch = H / 8;
  if (nch <= 64)
    hipLaunchKernelGGL((ln_bwd_dx_kernel<T, 1>), grid, blk, 0, st, (const T*)dy, (const T*)x, mean, rstd,
                       (const T*)g, (const T*)dres, (T*)dx, T_, H);
  else if (nch <= 256)
    hipLaunchKernelGGL((ln_bwd_dx_kernel<T, 4>), grid, blk, 0, st, (const T*)dy, (const T*)x, mean, rstd,
                       (const T*)g, (const T*)dres, (T*)dx, T_, H);
  else if (nch <= 512)
    hipLaunchKernelGGL((ln_bwd_dx_kernel<T, 8>), grid, blk, 0, st, (const T*)dy, (const T*)x, mean, rstd,
                       (const T*)g, (const T*)dres, (T*)dx, T_, H);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t layernorm_fwd(DType dt, const void* x, const void* g, const void* b, void* y, float* mean, float* rstd,
                         int T_, int H, float eps, hipStream_t st) {
  if (T_ <= 0) return hipSuccess;
  return dt == DT_BF16 ? ln_fwd_t<bf16>(x, g, b, y, mean, rstd, T_, H, eps, st)
                       : ln_fwd_t<float>(x, g, b, y, mean, rstd, T_, H, eps, st);
}

hipError_t layernorm_bwd_dx(DType dt, const void* dy, const void* x, const float* mean, const float* rstd,
                            const void* g, const void* dres, void* dx, int T_, int H, hipStream_t st) {
  if (T_ <= 0) return hipSuccess;
  return dt == DT_BF16 ? ln_bwd_t<bf16>(dy, x, mean, rstd, g, dres, dx, T_, H, st)
                       : ln_bwd_t<float>(dy, x, mean, rstd, g, dres, dx, T_, H, st);
}

// ---------------------------------------------------------------------------
// LayerNorm backward fused with the column sums that follow it.  Workgroup b
// of kLnBlocks takes rows [T b / kLnBlocks, T (b + 1) / kLnBlocks) (an even
// share, so the grid is one balanced round) across all H columns: wave w
// owns columns [512 w, 512 w + 512), eight per lane, so each row read is one
// contiguous 1 KB segment per wave.  Rows go four at a time; a row's two
// sums (of dxh and dxh * xh) are combined over the waves through LDS in wave
// order, then every lane finishes its columns of dx and adds, per column
// and in row order, dy * xh (the gain gradient), dy (the shift gradient) and
// optionally dx itself (the bias gradient of the layer that produced this
// LayerNorm's input).  The per-block sums go to partial [b][H] (fp32), which
// colsum_finish adds in block order: deterministic.  One pass reads dy, x
// (and dres) once, instead of once for dx and again for the column sums.
// ---------------------------------------------------------------------------
// (bf16: at most 128 registers, two workgroups per CU)
template <typename T, int R>
__global__ void __launch_bounds__(512, sizeof(T) == 2 ? 4 : 2)
    ln_bwd_fused_kernel(const T* dy, const T* x, const float* __restrict__ mean, const float* __restrict__ rstd,
                        const T* g, const T* dres, T* dx, int T_, int H, float* pg, float* pb, float* pout) {
  __shared__ float red[2][R][8][2];  // [batch parity][row][wave][sum]
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int col = w * 512 + lane * 8;
  const bool on = col < H;
  const int nw = (H + 511) / 512;  // waves holding columns
  const int r0 = (int)((long)T_ * blockIdx.x / kLnBlocks), r1 = (int)((long)T_ * (blockIdx.x + 1) / kLnBlocks);
  float gv[8], ag[8], ab[8], ao[8];
  {
    Vec8<T> gg;
    if (on) gg.load(g + col); else gg.zero();
#pragma unroll
    for (int e = 0; e < 8; ++e) { gv[e] = gg.get(e); ag[e] = 0.f; ab[e] = 0.f; ao[e] = 0.f; }
  }
  const float invH = 1.f / (float)H;
  // Two row batches in flight: batch i + 1 is loaded before batch i's
  // barrier, so its memory latency overlaps the barrier, the output and the
  // stores of batch i.
  Vec8<T> a[2][R], xx[2][R], rr[2][R];
  auto load = [&](int buf, int rb) {
#pragma unroll
    for (int u = 0; u < R; ++u) {
      const int r = rb + u;
      if (on && r < r1) {
        a[buf][u].load(dy + (long)r * H + col);
        xx[buf][u].load(x + (long)r * H + col);
        if (dres) rr[buf][u].load(dres + (long)r * H + col); else rr[buf][u].zero();
      } else {
        a[buf][u].zero(); xx[buf][u].zero(); rr[buf][u].zero();
      }
    }
  };
  auto batch = [&](auto bufc, int rb, int par) {
    constexpr int B = decltype(bufc)::value;
    float mu[R], rs[R], s1[R], s2[R];
#pragma unroll
    for (int u = 0; u < R; ++u) {
      const int r = rb + u;
      // row statistics: wave-uniform (scalar) loads, which do not queue
      // behind the vector stores of the previous batch
      mu[u] = r < r1 ? mean[r] : 0.f;
      rs[u] = r < r1 ? rstd[r] : 0.f;
      s1[u] = 0.f; s2[u] = 0.f;
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        const float xh = (xx[B][u].get(e) - mu[u]) * rs[u], d = a[B][u].get(e) * gv[e];
        s1[u] += d;
        s2[u] += d * xh;
      }
      s1[u] = wave_sum(s1[u]);
      s2[u] = wave_sum(s2[u]);
    }
    if (lane == 0) {
#pragma unroll
      for (int u = 0; u < R; ++u) { red[par][u][w][0] = s1[u]; red[par][u][w][1] = s2[u]; }
    }
    if (rb + R < r1) load(B ^ 1, rb + R);
    __syncthreads();  // one barrier per batch: the other parity's slots are free again
    // the packed rows are re-read from here on (values converted before the
    // barrier are not kept live across it)
#pragma unroll
    for (int u = 0; u < R; ++u) { a[B][u].settle(); xx[B][u].settle(); }
#pragma unroll
    for (int u = 0; u < R; ++u) {
      float t1 = 0.f, t2 = 0.f;
      for (int v = 0; v < nw; ++v) { t1 += red[par][u][v][0]; t2 += red[par][u][v][1]; }
      const float m1 = t1 * invH, m2 = t2 * invH;
      const int r = rb + u;
      if (on && r < r1) {
        float out[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float xh = (xx[B][u].get(e) - mu[u]) * rs[u], dv = a[B][u].get(e);
          out[e] = rr[B][u].get(e) + rs[u] * (dv * gv[e] - m1 - xh * m2);
          ag[e] += dv * xh;
          ab[e] += dv;
        }
        Vec8<T> o;
        o.set(out);
        o.store(dx + (long)r * H + col);
        if (pout) {
#pragma unroll
          for (int e = 0; e < 8; ++e) ao[e] += o.get(e);  // the stored (rounded) values
        }
      }
    }
  };
  load(0, r0);
  int par = 0;
  for (int rb = r0; rb < r1; rb += 2 * R) {
    batch(std::integral_constant<int, 0>{}, rb, par);
    par ^= 1;
    if (rb + R < r1) {
      batch(std::integral_constant<int, 1>{}, rb + R, par);
      par ^= 1;
    }
  }
  if (on) {
    const long base = (long)blockIdx.x * H + col;
    if (pg) {
      st16(pg + base, u32x4{__float_as_uint(ag[0]), __float_as_uint(ag[1]), __float_as_uint(ag[2]), __float_as_uint(ag[3])});
      st16(pg + base + 4, u32x4{__float_as_uint(ag[4]), __float_as_uint(ag[5]), __float_as_uint(ag[6]), __float_as_uint(ag[7])});
      st16(pb + base, u32x4{__float_as_uint(ab[0]), __float_as_uint(ab[1]), __float_as_uint(ab[2]), __float_as_uint(ab[3])});
      st16(pb + base + 4, u32x4{__float_as_uint(ab[4]), __float_as_uint(ab[5]), __float_as_uint(ab[6]), __float_as_uint(ab[7])});
    }
    if (pout) {
      st16(pout + base, u32x4{__float_as_uint(ao[0]), __float_as_uint(ao[1]), __float_as_uint(ao[2]), __float_as_uint(ao[3])});
      st16(pout + base + 4, u32x4{__float_as_uint(ao[4]), __float_as_uint(ao[5]), __float_as_uint(ao[6]), __float_as_uint(ao[7])});
    }
  }
}

hipError_t layernorm_bwd_fused(DType dt, const void* dy, const void* x, const float* mean, const float* rstd,
                               const void* g, const void* dres, void* dx, int T_, int H, float* pg, float* pb,
                               float* pout, hipStream_t st) {
  if (T_ <= 0) return hipSuccess;
  if (H > 4096 || H % 8 != 0 || (pg == nullptr) != (pb == nullptr)) return hipErrorInvalidValue;
  const dim3 grid((unsigned)kLnBlocks), blk(512);
  if (dt == DT_BF16) {
    hipLaunchKernelGGL((ln_bwd_fused_kernel<bf16, 2>), grid, blk, 0, st, (const bf16*)dy, (const bf16*)x, mean, rstd,
                       (const bf16*)g, (const bf16*)dres, (bf16*)dx, T_, H, pg, pb, pout);
  } else {
    hipLaunchKernelGGL((ln_bwd_fused_kernel<float, 2>), grid, blk, 0, st, (const float*)dy, (const float*)x, mean,
                       rstd, (const float*)g, (const float*)dres, (float*)dx, T_, H, pg, pb, pout);
  }
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Column sums.  Workgroup (cb, rb): columns cb*512 .. +511 (8 per lane), rows
// rb*kColsumRows .. ; wave w takes every 4th row; the four waves combine in
// LDS in a fixed order.
// ---------------------------------------------------------------------------
template <typename T, int MODE>
__global__ void __launch_bounds__(256) colsum_partial_kernel(const T* X, long ldx, const T* Y, const float* mean,
                                                             const float* rstd, int T_, int N, float* part,
                                                             float* part2) {
  __shared__ float sh[2][4][512];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int col = blockIdx.x * 512 + lane * 8;
  const int r0 = blockIdx.y * kColsumRows;
  const int r1 = min(r0 + kColsumRows, T_);
  float a1[8], a2[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) { a1[e] = 0.f; a2[e] = 0.f; }
  // rows r0 + w, r0 + w + 4, ... in order; eight of them loaded before any
  // is added, so each wave keeps eight loads in flight (same summation order)
  auto add = [&](const Vec8<T>& xv, const Vec8<T>& yv, int r) {
    if constexpr (MODE == 0) {
#pragma unroll
      for (int e = 0; e < 8; ++e) a1[e] += xv.get(e);
    } else {
      const float mu = mean[r], rs = rstd[r];
#pragma unroll
      for (int e = 0; e < 8; ++e) {
        a1[e] += xv.get(e) * ((yv.get(e) - mu) * rs);
        a2[e] += xv.get(e);
      }
    }
  };
  if (col < N) {
    int r = r0 + w;
    constexpr int B = MODE == 0 ? 8 : 4;
    for (; r + 4 * (B - 1) < r1; r += 4 * B) {
      Vec8<T> xv[B], yv[B];
#pragma unroll
      for (int u = 0; u < B; ++u) {
        xv[u].load(X + (long)(r + 4 * u) * ldx + col);
        if constexpr (MODE == 1) yv[u].load(Y + (long)(r + 4 * u) * ldx + col);
      }
#pragma unroll
      for (int u = 0; u < B; ++u) add(xv[u], yv[u], r + 4 * u);
    }
    for (; r < r1; r += 4) {
      Vec8<T> xv, yv;
      xv.load(X + (long)r * ldx + col);
      if constexpr (MODE == 1) yv.load(Y + (long)r * ldx + col);
      add(xv, yv, r);
    }
  }
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    sh[0][w][lane * 8 + e] = a1[e];
    sh[1][w][lane * 8 + e] = a2[e];
  }
  __syncthreads();
  for (int c = threadIdx.x; c < 512; c += 256) {
    const int n = blockIdx.x * 512 + c;
    if (n < N) {
      part[(long)blockIdx.y * N + n] = ((sh[0][0][c] + sh[0][1][c]) + sh[0][2][c]) + sh[0][3][c];
      if constexpr (MODE == 1)
        part2[(long)blockIdx.y * N + n] = ((sh[1][0][c] + sh[1][1][c]) + sh[1][2][c]) + sh[1][3][c];
    }
  }
}

hipError_t colsum_partial(DType dt, int mode, const void* X, long ldx, const void* Y, const float* mean,
                          const float* rstd, int T_, int N, float* part, float* part2, hipStream_t st) {
  if (T_ <= 0 || N <= 0) return hipSuccess;
  dim3 grid((N + 511) / 512, colsum_blocks(T_)), blk(256);
  if (dt == DT_BF16) {
    if (mode == 0)
      hipLaunchKernelGGL((colsum_partial_kernel<bf16, 0>), grid, blk, 0, st, (const bf16*)X, ldx, (const bf16*)Y,
                         mean, rstd, T_, N, part, part2);
    else
      hipLaunchKernelGGL((colsum_partial_kernel<bf16, 1>), grid, blk, 0, st, (const bf16*)X, ldx, (const bf16*)Y,
                         mean, rstd, T_, N, part, part2);
  } else {
    if (mode == 0)
      hipLaunchKernelGGL((colsum_partial_kernel<float, 0>), grid, blk, 0, st, (const float*)X, ldx,
                         (const float*)Y, mean, rstd, T_, N, part, part2);
    else
      hipLaunchKernelGGL((colsum_partial_kernel<float, 1>), grid, blk, 0, st, (const float*)X, ldx,
                         (const float*)Y, mean, rstd, T_, N, part, part2);
  }
  return hipGetLastError();
}

// out[n] += sum over the nblk partial rows.  A workgroup takes 64 columns;
// its 16 waves sum contiguous sixteenths of the rows (eight loads in flight
// per lane), and the sixteenths are added in order through LDS: a fixed
// order, so the result is deterministic.  Up to three (partial, out) pairs
// of one shape go in one launch (grid y).
struct FinishSet {
  const float* part[3];
  float* out[3];
};
__global__ void __launch_bounds__(1024) colsum_finish_kernel(FinishSet fs, int nblk, int N) {
  constexpr int NW = 16;
  __shared__ float q[NW][64];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int n = blockIdx.x * 64 + lane;
  const float* part = fs.part[blockIdx.y];
  const int per = (nblk + NW - 1) / NW;
  const int b0 = min(nblk, w * per), b1 = min(nblk, b0 + per);
  float s = 0.f;
  if (n < N) {
    int b = b0;
    for (; b + 8 <= b1; b += 8) {
      float v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) v[u] = part[(long)(b + u) * N + n];
#pragma unroll
      for (int u = 0; u < 8; ++u) s += v[u];
    }
    for (; b < b1; ++b) s += part[(long)b * N + n];
  }
  q[w][lane] = s;
  __syncthreads();
  if (w == 0 && n < N) {
    float t = q[0][lane];
#pragma unroll
    for (int v = 1; v < NW; ++v) t += q[v][lane];
    fs.out[blockIdx.y][n] += t;
  }
}

hipError_t colsum_finish_n(const float* const* parts, float* const* outs, int count, int nblk, int N,
                           hipStream_t st) {
  if (N <= 0 || count <= 0) return hipSuccess;
  if (count > 3) return hipErrorInvalidValue;
  FinishSet fs{};
  for (int i = 0; i < count; ++i) { fs.part[i] = parts[i]; fs.out[i] = outs[i]; }
  hipLaunchKernelGGL(colsum_finish_kernel, dim3((N + 63) / 64, count), dim3(1024), 0, st, fs, nblk, N);
  return hipGetLastError();
}

hipError_t colsum_finish(const float* part, int nblk, int N, float* out, hipStream_t st) {
  return colsum_finish_n(&part, &out, 1, nblk, N, st);
}

// ---------------------------------------------------------------------------
// Client packing (byte copies, 16-byte vectors).
// ---------------------------------------------------------------------------
__global__ void pack_client_kernel(const char* client, char* packed, const int32_t* cu, int s0, int nseq,
                                   int row_bytes, bool unpack) {
  const int p = blockIdx.x, b = blockIdx.y;
  const int s = s0 + b;
  const int r0 = cu[s], L = cu[s + 1] - r0;
  const long crow = ((long)p * nseq + b) * row_bytes;
  const long prow = (long)(r0 + p) * row_bytes;
  for (int o = threadIdx.x * 16; o < row_bytes; o += blockDim.x * 16) {
    if (p < L) {
      if (unpack) st16((void*)(const_cast<char*>(client) + crow + o), ld16(packed + prow + o));
      else st16(packed + prow + o, ld16(client + crow + o));
    } else if (unpack) {
      st16((void*)(const_cast<char*>(client) + crow + o), u32x4{0, 0, 0, 0});
    }
  }
}

hipError_t pack_client(DType dt, const void* client, void* packed, const int32_t* cu, int s0, int nseq, int Lmax,
                       int H, bool unpack, hipStream_t st) {
  if (Lmax <= 0 || nseq <= 0) return hipSuccess;
  const int row_bytes = H * (dt == DT_BF16 ? 2 : 4);
  hipLaunchKernelGGL(pack_client_kernel, dim3(Lmax, nseq), dim3(128), 0, st, (const char*)client, (char*)packed,
                     cu, s0, nseq, row_bytes, unpack);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// P-tuning v2 prefix gradients: out_k[e] += sum_s part[0][s][e], out_v[e] +=
// sum_s part[1][s][e] over e < n (n = num_prefix * hidden), sequences in
// index order (deterministic).  Four elements per thread.
// ---------------------------------------------------------------------------
__global__ void prefix_grad_reduce_kernel(const float* part, int S, long n, float* out_k, float* out_v) {
  const long e = ((long)blockIdx.x * blockDim.x + threadIdx.x) * 4;
  const int which = blockIdx.y;
  if (e >= n) return;
  const float* src = part + (long)which * S * n + e;
  float* dst = (which ? out_v : out_k) + e;
  Vec4<float> acc;
  acc.load(dst);
  float a[4] = {acc.get(0), acc.get(1), acc.get(2), acc.get(3)};
  for (int s = 0; s < S; ++s) {
    Vec4<float> v;
    v.load(src + (long)s * n);
#pragma unroll
    for (int i = 0; i < 4; ++i) a[i] += v.get(i);
  }
  acc.set(a);
  acc.store(dst);
}

hipError_t prefix_grad_reduce(const float* part, int S, long n, float* out_k, float* out_v, hipStream_t st) {
  if (n <= 0) return hipSuccess;
  const dim3 g((unsigned)((n / 4 + 255) / 256), 2);
  hipLaunchKernelGGL(prefix_grad_reduce_kernel, g, dim3(256), 0, st, part, S, n, out_k, out_v);
  return hipGetLastError();
}

}  // namespace flglm
