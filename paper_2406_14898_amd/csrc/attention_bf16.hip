// bf16 attention over packed ragged sequences for gfx950 (the fp32 debug
// mode uses attention.hip).  Same contract as attention.hip: every
// workgroup stays inside one (sequence, head); key j is visible to query i
// iff j <= max(i, P - 1); scale 1/sqrt(d) (Appendix A: softmax(QK^T/sqrt(d_h))).
//
// Data movement:
//   * K, V (forward, dq) and Q, dO (dk/dv) tiles of 64 rows x d go from HBM
//     straight into LDS with buffer loads in LDS-DMA mode, double-buffered:
//     the next tile streams in while the current one is used.  Buffer
//     resources are bounded at the sequence end, so rows past it read as
//     zero.
//   * Tiles stay in their global layout ([row][d], 16-byte chunks swizzled
//     by chunk ^ 2 (row & 7) for d = 128, chunk ^ (row & 7) for d = 64).
//     Operands whose contraction runs along the feature dimension use
//     16-byte reads; operands contracted along the rows (V^T, K^T, Q^T,
//     dO^T) use transpose reads (ds_read_b64_tr_b16).  For 256-byte rows this
//     swizzle keeps both kinds free of LDS bank conflicts (measured).
//   * The probabilities never touch LDS: scores are computed transposed so
//     that two adjacent 16-row result tiles hold, per lane, exactly the eight
//     reduction slots {4g .. 4g+3, 16+4g .. 16+4g+3} of the next product, and
//     the transpose reads of the other operand are issued with that slot
//     order (rows kb + 4g + e and kb + 16 + 4g + e).
// Kernels: forward (S^T = K Q^T, online softmax, O^T += V^T P^T); dq
// (S^T, dP^T = V dO^T, dQ^T += K^T dS^T); dk/dv (S = Q K^T, dP = dO V^T,
// dV^T += dO^T P, dK^T += Q^T dS).  Every output element has one writer.
#include "common.h"
#include "kernels.h"

namespace flglm {
namespace {

constexpr int kRows = 64;  // rows per LDS tile
typedef short i16x4 __attribute__((ext_vector_type(4)));
#define LDS_AS __attribute__((address_space(3)))

struct SeqB {
  int r0, L, P;
};
__device__ __forceinline__ SeqB seqb(const int32_t* cu, const int32_t* prefix, int s) {
  SeqB si;
  si.r0 = cu[s];
  si.L = cu[s + 1] - si.r0;
  si.P = prefix ? prefix[s] : 0;
  return si;
}
__device__ __forceinline__ bool vis(int i, int j, int L, int P) { return j < L && (j <= i || j < P); }

template <int D>
__device__ __forceinline__ int swz(int row) {
  return D == 128 ? 2 * (row & 7) : (row & 7);
}

// DMA a [64 rows][D] tile: rows row0 .. of the resource (row stride ld
// elements) into LDS at byte address tile; D/8 instructions per tile,
// spread over the 4 waves.
template <int D>
__device__ __forceinline__ void dma_tile(i32x4 rs, long ld, int row0, uint32_t tile, int wave, int lane) {
  constexpr int CH = D / 8;          // chunks per row
  constexpr int RPI = 64 / CH;       // rows per instruction
#pragma unroll
  for (int i = 0; i < CH / 4; ++i) {
    const int inst = i * 4 + wave;
    const int row = inst * RPI + lane / CH;
    const int q = (lane % CH) ^ swz<D>(row);
    const uint32_t voff = (uint32_t)((long)(row0 + row) * ld + q * 8) * 2u;
    dma_lds<16>(rs, tile + inst * 1024, voff);
  }
}

// 16 rows (r0 + fr) x reduction slots 32c + 8g .. +7 (16-byte read).
template <int D>
__device__ __forceinline__ bf16x8 frag_row(const bf16* tile, int r0, int c, int fr, int fg) {
  const int row = r0 + fr;
  return __builtin_bit_cast(bf16x8, ld16(tile + row * D + (((4 * c + fg) ^ swz<D>(row)) * 8)));
}
// Columns d0 + j (lane j of the group) x reduction rows
// {kb + 4g + e, kb + 16 + 4g + e}, e < 4 (two transpose reads).
template <int D>
__device__ __forceinline__ bf16x8 frag_tr(const bf16* tile, int kb, int d0, int fr, int fg) {
  const int col = d0 + 4 * (fr & 3);
  const int r1 = kb + 4 * fg + (fr >> 2), r2 = r1 + 16;
  const bf16* p1 = tile + r1 * D + (((col >> 3) ^ swz<D>(r1)) * 8) + (col & 7);
  const bf16* p2 = tile + r2 * D + (((col >> 3) ^ swz<D>(r2)) * 8) + (col & 7);
  i16x4 a = __builtin_amdgcn_ds_read_tr16_b64_v4i16((LDS_AS i16x4*)p1);
  i16x4 b = __builtin_amdgcn_ds_read_tr16_b64_v4i16((LDS_AS i16x4*)p2);
  return __builtin_bit_cast(bf16x8, __builtin_shufflevector(a, b, 0, 1, 2, 3, 4, 5, 6, 7));
}

__device__ __forceinline__ bf16x8 pack_p(const float (&x)[4], const float (&y)[4]) {
  return bf16x8{from_f32<bf16>(x[0]), from_f32<bf16>(x[1]), from_f32<bf16>(x[2]), from_f32<bf16>(x[3]),
                from_f32<bf16>(y[0]), from_f32<bf16>(y[1]), from_f32<bf16>(y[2]), from_f32<bf16>(y[3])};
}

__device__ __forceinline__ void bar() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Inverse rotation of a gradient held as lane tiles acc[dt] (rows d = 16dt +
// 4g + i): pairs (d, d + r/2) for d < r/2, angle -p*theta.
template <int D>
__device__ __forceinline__ void rope_back(f32x4 (&acc)[D / 16], int p, int r, int fg, const float* ct,
                                          const float* stb) {
  const int half = r / 2, ht = half / 16;
#pragma unroll
  for (int dt = 0; dt < D / 16; ++dt) {
    if (dt < ht) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int di = 16 * dt + 4 * fg + i;
        const float c = ct[(long)p * half + di], sn = stb[(long)p * half + di];
        const float x1 = acc[dt][i], x2 = acc[dt + ht][i];
        acc[dt][i] = x1 * c + x2 * sn;
        acc[dt + ht][i] = x2 * c - x1 * sn;
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Forward: 128 queries per workgroup (4 waves x 32), key tiles of 64.
// ---------------------------------------------------------------------------
template <int D>
__global__ void __launch_bounds__(256) fwd_kernel(AttnDesc a) {
  constexpr int NC = D / 32, QS = 2, BM = 128;
  __shared__ __attribute__((aligned(1024))) bf16 Ks[2][kRows * D];
  __shared__ __attribute__((aligned(1024))) bf16 Vs[2][kRows * D];

  const int s = blockIdx.z, h = blockIdx.y;
  const int q0 = (gridDim.x - 1 - blockIdx.x) * BM;  // longest-running query tiles first
  const SeqB si = seqb(a.cu_seqlens, a.prefix_len, s);
  if (q0 >= si.L) return;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int fr = lane & 15, fg = lane >> 4;
  const bf16* qkv = static_cast<const bf16*>(a.qkv);
  const long ld = a.ld_qkv;
  const int H = a.hidden;
  const float sl2 = kLog2e / sqrtf((float)D);

  const uint32_t seq_bytes = (uint32_t)((long)si.L * ld * 2);
  const auto rk = buf_rsrc(qkv + (long)si.r0 * ld + H + h * D, seq_bytes);
  const auto rv = buf_rsrc(qkv + (long)si.r0 * ld + 2 * H + h * D, seq_bytes);
  const int kv_end = min(si.L, max(q0 + BM, si.P));
  const int nkt = (kv_end + kRows - 1) / kRows;
  const uint32_t lds_k = FL_LDS_ADDR(&Ks[0][0]), lds_v = FL_LDS_ADDR(&Vs[0][0]);
  auto issue = [&](int kt) {
    dma_tile<D>(rk, ld, kt * kRows, lds_k + (kt & 1) * (kRows * D * 2), w, lane);
    dma_tile<D>(rv, ld, kt * kRows, lds_v + (kt & 1) * (kRows * D * 2), w, lane);
  };
  issue(0);

  bf16x8 qf[QS][NC];
#pragma unroll
  for (int qs = 0; qs < QS; ++qs) {
    const int qi = q0 + 32 * w + 16 * qs + fr;
#pragma unroll
    for (int c = 0; c < NC; ++c)
      qf[qs][c] = qi < si.L ? __builtin_bit_cast(bf16x8, ld16(qkv + (long)(si.r0 + qi) * ld + h * D + 32 * c + 8 * fg))
                            : bf16x8{};
  }
#pragma unroll
  for (int qs = 0; qs < QS; ++qs)
#pragma unroll
    for (int c = 0; c < NC; ++c) settle(qf[qs][c]);
  f32x4 acc[D / 16][QS];
#pragma unroll
  for (int dt = 0; dt < D / 16; ++dt)
#pragma unroll
    for (int qs = 0; qs < QS; ++qs) acc[dt][qs] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m[QS], l[QS];
#pragma unroll
  for (int qs = 0; qs < QS; ++qs) { m[qs] = -INFINITY; l[qs] = 0.f; }

  for (int kt = 0; kt < nkt; ++kt) {
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    bar();  // tile kt landed for every wave; slot (kt+1)&1 is free
    if (kt + 1 < nkt) issue(kt + 1);
    const bf16* ks = Ks[kt & 1];
    const bf16* vs = Vs[kt & 1];
    const int j0 = kt * kRows;

    f32x4 st[QS][4];
#pragma unroll
    for (int qs = 0; qs < QS; ++qs)
#pragma unroll
      for (int at = 0; at < 4; ++at) st[qs][at] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      bf16x8 kf[4];
#pragma unroll
      for (int at = 0; at < 4; ++at) kf[at] = frag_row<D>(ks, 16 * at, c, fr, fg);
#pragma unroll
      for (int qs = 0; qs < QS; ++qs)
#pragma unroll
        for (int at = 0; at < 4; ++at) st[qs][at] = mma16(kf[at], qf[qs][c], st[qs][at]);
    }
    float p[QS][4][4];
#pragma unroll
    for (int qs = 0; qs < QS; ++qs) {
      const int qi = q0 + 32 * w + 16 * qs + fr;
      float mx = -INFINITY;
#pragma unroll
      for (int at = 0; at < 4; ++at)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int j = j0 + 16 * at + 4 * fg + i;
          const float v = vis(qi, j, si.L, si.P) ? st[qs][at][i] * sl2 : -INFINITY;
          p[qs][at][i] = v;
          mx = fmaxf(mx, v);
        }
      mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
      mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
      const float mnew = fmaxf(m[qs], mx);
      const float alpha = (mnew == -INFINITY) ? 1.f : exp2f(m[qs] - mnew);
      m[qs] = mnew;
      float ls = 0.f;
#pragma unroll
      for (int at = 0; at < 4; ++at)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float e = (p[qs][at][i] == -INFINITY) ? 0.f : exp2f(p[qs][at][i] - mnew);
          p[qs][at][i] = e;
          ls += e;
        }
      l[qs] = l[qs] * alpha + ls;
#pragma unroll
      for (int dt = 0; dt < D / 16; ++dt) acc[dt][qs] *= alpha;
    }
#pragma unroll
    for (int c2 = 0; c2 < 2; ++c2) {
      bf16x8 pf[QS];
#pragma unroll
      for (int qs = 0; qs < QS; ++qs) pf[qs] = pack_p(p[qs][2 * c2], p[qs][2 * c2 + 1]);
#pragma unroll
      for (int dt = 0; dt < D / 16; ++dt) {
        const bf16x8 vf = frag_tr<D>(vs, 32 * c2, 16 * dt, fr, fg);
#pragma unroll
        for (int qs = 0; qs < QS; ++qs) acc[dt][qs] = mma16(vf, pf[qs], acc[dt][qs]);
      }
    }
  }

  bf16* o = static_cast<bf16*>(a.o);
#pragma unroll
  for (int qs = 0; qs < QS; ++qs) {
    float lt = l[qs];
    lt += __shfl_xor(lt, 16, 64);
    lt += __shfl_xor(lt, 32, 64);
    const int qi = q0 + 32 * w + 16 * qs + fr;
    if (qi >= si.L) continue;
    const float inv = 1.f / lt;
#pragma unroll
    for (int dt = 0; dt < D / 16; ++dt) {
      const float v[4] = {acc[dt][qs][0] * inv, acc[dt][qs][1] * inv, acc[dt][qs][2] * inv, acc[dt][qs][3] * inv};
      Vec4<bf16> ov;
      ov.set(v);
      ov.store(o + (long)(si.r0 + qi) * a.ld_o + h * D + 16 * dt + 4 * fg);
    }
    if (fg == 0) a.lse[(long)(si.r0 + qi) * a.num_heads + h] = m[qs] * 0.69314718055994531f + logf(lt);
  }
}

// ---------------------------------------------------------------------------
// Backward, dq: 64 queries per workgroup (4 waves x 16), key tiles of 64.
// ---------------------------------------------------------------------------
template <int D>
__global__ void __launch_bounds__(256) dq_kernel(AttnDesc a) {
  constexpr int NC = D / 32, BM = 64;
  __shared__ __attribute__((aligned(1024))) bf16 Ks[2][kRows * D];
  __shared__ __attribute__((aligned(1024))) bf16 Vs[2][kRows * D];

  const int s = blockIdx.z, h = blockIdx.y;
  const int q0 = (gridDim.x - 1 - blockIdx.x) * BM;
  const SeqB si = seqb(a.cu_seqlens, a.prefix_len, s);
  if (q0 >= si.L) return;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int fr = lane & 15, fg = lane >> 4;
  const bf16* qkv = static_cast<const bf16*>(a.qkv);
  const bf16* dout = static_cast<const bf16*>(a.dout);
  const long ld = a.ld_qkv;
  const int H = a.hidden;
  const float sl2 = kLog2e / sqrtf((float)D);

  const uint32_t seq_bytes = (uint32_t)((long)si.L * ld * 2);
  const auto rk = buf_rsrc(qkv + (long)si.r0 * ld + H + h * D, seq_bytes);
  const auto rv = buf_rsrc(qkv + (long)si.r0 * ld + 2 * H + h * D, seq_bytes);
  const int kv_end = min(si.L, max(q0 + BM, si.P));
  const int nkt = (kv_end + kRows - 1) / kRows;
  const uint32_t lds_k = FL_LDS_ADDR(&Ks[0][0]), lds_v = FL_LDS_ADDR(&Vs[0][0]);
  auto issue = [&](int kt) {
    dma_tile<D>(rk, ld, kt * kRows, lds_k + (kt & 1) * (kRows * D * 2), w, lane);
    dma_tile<D>(rv, ld, kt * kRows, lds_v + (kt & 1) * (kRows * D * 2), w, lane);
  };
  issue(0);

  const int qi = q0 + 16 * w + fr;
  const bool qvalid = qi < si.L;
  bf16x8 qf[NC], dof[NC];
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    qf[c] = qvalid ? __builtin_bit_cast(bf16x8, ld16(qkv + (long)(si.r0 + qi) * ld + h * D + 32 * c + 8 * fg))
                   : bf16x8{};
    dof[c] = qvalid ? __builtin_bit_cast(bf16x8,
                                         ld16(dout + (long)(si.r0 + qi) * a.ld_dout + h * D + 32 * c + 8 * fg))
                    : bf16x8{};
  }
  const float lse2 = qvalid ? a.lse[(long)(si.r0 + qi) * a.num_heads + h] * kLog2e : 0.f;
  float dlt = qvalid ? a.delta[(long)(si.r0 + qi) * a.num_heads + h] : 0.f;
  float lse2s = lse2;
#pragma unroll
  for (int c = 0; c < NC; ++c) { settle(qf[c]); settle(dof[c]); }
  settle(dlt);
  settle(lse2s);
  f32x4 acc[D / 16];
#pragma unroll
  for (int dt = 0; dt < D / 16; ++dt) acc[dt] = f32x4{0.f, 0.f, 0.f, 0.f};

  for (int kt = 0; kt < nkt; ++kt) {
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    bar();
    if (kt + 1 < nkt) issue(kt + 1);
    const bf16* ks = Ks[kt & 1];
    const bf16* vs = Vs[kt & 1];
    const int j0 = kt * kRows;
    f32x4 st[4], dp[4];
#pragma unroll
    for (int at = 0; at < 4; ++at) { st[at] = f32x4{0.f, 0.f, 0.f, 0.f}; dp[at] = st[at]; }
#pragma unroll
    for (int c = 0; c < NC; ++c) {
#pragma unroll
      for (int at = 0; at < 4; ++at) {
        st[at] = mma16(frag_row<D>(ks, 16 * at, c, fr, fg), qf[c], st[at]);
        dp[at] = mma16(frag_row<D>(vs, 16 * at, c, fr, fg), dof[c], dp[at]);
      }
    }
    float ds[4][4];
#pragma unroll
    for (int at = 0; at < 4; ++at)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int j = j0 + 16 * at + 4 * fg + i;
        const float pr = (qvalid && vis(qi, j, si.L, si.P)) ? exp2f(st[at][i] * sl2 - lse2s) : 0.f;
        ds[at][i] = pr * (dp[at][i] - dlt);
      }
#pragma unroll
    for (int c2 = 0; c2 < 2; ++c2) {
      const bf16x8 df = pack_p(ds[2 * c2], ds[2 * c2 + 1]);
#pragma unroll
      for (int dt = 0; dt < D / 16; ++dt) acc[dt] = mma16(frag_tr<D>(ks, 32 * c2, 16 * dt, fr, fg), df, acc[dt]);
    }
  }
  if (!qvalid) return;
  const float sc = 1.f / sqrtf((float)D);
#pragma unroll
  for (int dt = 0; dt < D / 16; ++dt) acc[dt] *= sc;
  rope_back<D>(acc, qi, a.rotary_dim, fg, a.cos_t, a.sin_t);
  bf16* dq = static_cast<bf16*>(a.dqkv) + (long)(si.r0 + qi) * a.ld_dqkv + h * D;
#pragma unroll
  for (int dt = 0; dt < D / 16; ++dt) {
    const float v[4] = {acc[dt][0], acc[dt][1], acc[dt][2], acc[dt][3]};
    Vec4<bf16> ov;
    ov.set(v);
    ov.store(dq + 16 * dt + 4 * fg);
  }
}

// ---------------------------------------------------------------------------
// Backward, dk and dv: 64 keys per workgroup (4 waves x 16), query tiles of
// 64 with their LSE and delta rows.
// ---------------------------------------------------------------------------
template <int D>
__global__ void __launch_bounds__(256) dkdv_kernel(AttnDesc a) {
  constexpr int NC = D / 32, BK = 64;
  __shared__ __attribute__((aligned(1024))) bf16 Qs[2][kRows * D];
  __shared__ __attribute__((aligned(1024))) bf16 Os[2][kRows * D];
  __shared__ __attribute__((aligned(256))) float Ls[2][kRows];
  __shared__ __attribute__((aligned(256))) float Ds[2][kRows];

  const int s = blockIdx.z, h = blockIdx.y;
  const int k0 = (gridDim.x - 1 - blockIdx.x) * BK;
  const SeqB si = seqb(a.cu_seqlens, a.prefix_len, s);
  if (k0 >= si.L) return;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int fr = lane & 15, fg = lane >> 4;
  const bf16* qkv = static_cast<const bf16*>(a.qkv);
  const bf16* dout = static_cast<const bf16*>(a.dout);
  const long ld = a.ld_qkv;
  const int H = a.hidden, nh = a.num_heads;
  const float sl2 = kLog2e / sqrtf((float)D);

  const auto rq = buf_rsrc(qkv + (long)si.r0 * ld + h * D, (uint32_t)((long)si.L * ld * 2));
  const auto ro = buf_rsrc(dout + (long)si.r0 * a.ld_dout + h * D, (uint32_t)((long)si.L * a.ld_dout * 2));
  const auto rl = buf_rsrc(a.lse + (long)si.r0 * nh + h, (uint32_t)((long)si.L * nh * 4 - h * 4));
  const auto rd = buf_rsrc(a.delta + (long)si.r0 * nh + h, (uint32_t)((long)si.L * nh * 4 - h * 4));
  const int qstart = ((k0 < si.P) ? 0 : k0) / kRows;
  const int nqt = (si.L + kRows - 1) / kRows;
  const uint32_t lds_q = FL_LDS_ADDR(&Qs[0][0]), lds_o = FL_LDS_ADDR(&Os[0][0]);
  const uint32_t lds_l = FL_LDS_ADDR(&Ls[0][0]), lds_d = FL_LDS_ADDR(&Ds[0][0]);
  auto issue = [&](int qt) {
    const int slot = qt & 1;
    dma_tile<D>(rq, ld, qt * kRows, lds_q + slot * (kRows * D * 2), w, lane);
    dma_tile<D>(ro, a.ld_dout, qt * kRows, lds_o + slot * (kRows * D * 2), w, lane);
    // LSE (scaled on use) and delta rows: 64 x 4 bytes each
    const uint32_t voff = (uint32_t)((qt * kRows + lane) * nh) * 4u;
    if (w == 0) dma_lds<4>(rl, lds_l + slot * (kRows * 4), voff);
    if (w == 1) dma_lds<4>(rd, lds_d + slot * (kRows * 4), voff);
  };
  issue(qstart);

  const int kj = k0 + 16 * w + fr;
  const bool kvalid = kj < si.L;
  bf16x8 kf[NC], vf[NC];
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    kf[c] = kvalid ? __builtin_bit_cast(bf16x8, ld16(qkv + (long)(si.r0 + kj) * ld + H + h * D + 32 * c + 8 * fg))
                   : bf16x8{};
    vf[c] = kvalid
                ? __builtin_bit_cast(bf16x8, ld16(qkv + (long)(si.r0 + kj) * ld + 2 * H + h * D + 32 * c + 8 * fg))
                : bf16x8{};
  }
#pragma unroll
  for (int c = 0; c < NC; ++c) { settle(kf[c]); settle(vf[c]); }
  f32x4 dk[D / 16], dv[D / 16];
#pragma unroll
  for (int dt = 0; dt < D / 16; ++dt) { dk[dt] = f32x4{0.f, 0.f, 0.f, 0.f}; dv[dt] = dk[dt]; }

  for (int qt = qstart; qt < nqt; ++qt) {
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    bar();
    if (qt + 1 < nqt) issue(qt + 1);
    const bf16* qs_ = Qs[qt & 1];
    const bf16* os_ = Os[qt & 1];
    const float* ls_ = Ls[qt & 1];
    const float* dls = Ds[qt & 1];
    const int qb = qt * kRows;
    float pr[4][4], ds[4][4];
#pragma unroll
    for (int qs = 0; qs < 4; ++qs) {
      f32x4 st = f32x4{0.f, 0.f, 0.f, 0.f}, dp = st;
#pragma unroll
      for (int c = 0; c < NC; ++c) {
        st = mma16(frag_row<D>(qs_, 16 * qs, c, fr, fg), kf[c], st);
        dp = mma16(frag_row<D>(os_, 16 * qs, c, fr, fg), vf[c], dp);
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int ql = 16 * qs + 4 * fg + i;
        const int q = qb + ql;
        const float p = (kvalid && vis(q, kj, si.L, si.P)) ? exp2f(st[i] * sl2 - ls_[ql] * kLog2e) : 0.f;
        pr[qs][i] = p;
        ds[qs][i] = p * (dp[i] - dls[ql]);
      }
    }
#pragma unroll
    for (int c2 = 0; c2 < 2; ++c2) {
      const bf16x8 pf = pack_p(pr[2 * c2], pr[2 * c2 + 1]);
      const bf16x8 df = pack_p(ds[2 * c2], ds[2 * c2 + 1]);
#pragma unroll
      for (int dt = 0; dt < D / 16; ++dt) {
        dv[dt] = mma16(frag_tr<D>(os_, 32 * c2, 16 * dt, fr, fg), pf, dv[dt]);
        dk[dt] = mma16(frag_tr<D>(qs_, 32 * c2, 16 * dt, fr, fg), df, dk[dt]);
      }
    }
  }
  if (!kvalid) return;
  const float sc = 1.f / sqrtf((float)D);
#pragma unroll
  for (int dt = 0; dt < D / 16; ++dt) dk[dt] *= sc;
  rope_back<D>(dk, kj, a.rotary_dim, fg, a.cos_t, a.sin_t);
  bf16* row = static_cast<bf16*>(a.dqkv) + (long)(si.r0 + kj) * a.ld_dqkv + h * D;
#pragma unroll
  for (int dt = 0; dt < D / 16; ++dt) {
    const float vk[4] = {dk[dt][0], dk[dt][1], dk[dt][2], dk[dt][3]};
    const float vv[4] = {dv[dt][0], dv[dt][1], dv[dt][2], dv[dt][3]};
    Vec4<bf16> ok, ov;
    ok.set(vk);
    ov.set(vv);
    ok.store(row + H + 16 * dt + 4 * fg);
    ov.store(row + 2 * H + 16 * dt + 4 * fg);
  }
}

template <int D>
hipError_t fwd_launch(const AttnDesc& a, hipStream_t st) {
  dim3 grid((a.max_seqlen + 127) / 128, a.num_heads, a.num_seqs);
  hipLaunchKernelGGL((fwd_kernel<D>), grid, dim3(256), 0, st, a);
  return hipGetLastError();
}

template <int D>
hipError_t bwd_launch(const AttnDesc& a, hipStream_t st) {
  hipError_t e = attn_delta(DT_BF16, a, st);
  if (e != hipSuccess) return e;
  dim3 grid((a.max_seqlen + 63) / 64, a.num_heads, a.num_seqs);
  hipLaunchKernelGGL((dkdv_kernel<D>), grid, dim3(256), 0, st, a);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  hipLaunchKernelGGL((dq_kernel<D>), grid, dim3(256), 0, st, a);
  return hipGetLastError();
}

}  // namespace

// Byte offsets inside one sequence stay below 2^32 for the buffer resources.
bool attn_bf16_ok(const AttnDesc& a) {
  const long ld = a.ld_qkv > a.ld_dout ? a.ld_qkv : a.ld_dout;
  return (a.head_dim == 64 || a.head_dim == 128) && (long)a.max_seqlen * ld * 2 < (1L << 31);
}

hipError_t attn_fwd_bf16(const AttnDesc& a, hipStream_t st) {
  if (a.num_seqs <= 0 || a.max_seqlen <= 0) return hipSuccess;
  return a.head_dim == 128 ? fwd_launch<128>(a, st) : fwd_launch<64>(a, st);
}

hipError_t attn_bwd_bf16(const AttnDesc& a, hipStream_t st) {
  if (a.num_seqs <= 0 || a.max_seqlen <= 0) return hipSuccess;
  return a.head_dim == 128 ? bwd_launch<128>(a, st) : bwd_launch<64>(a, st);
}

}  // namespace flglm
