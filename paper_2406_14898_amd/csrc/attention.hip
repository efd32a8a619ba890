// Attention over packed ragged sequences, matrix-core tiles, fp32 softmax:
// the fp32 debug mode's kernels (bf16 runs on attention_bf16.hip).
//
// Every workgroup works inside one (sequence, head): its row range comes
// from cu_seqlens, so no score ever crosses a sequence (hence a client)
// boundary.  Mask: key j is visible to query i iff j <= max(i, P - 1), with P
// the bidirectional prefix of the sequence (P = 0 gives the causal mask).
// The softmax scale is 1/sqrt(d) (Appendix A writes softmax(QK^T/sqrt(d_h))).
//
// Layout trick shared by all three kernels: the matrix-core result tile puts
// one column per lane and four consecutive rows per lane group, so scores
// are computed with the dimension that the *next* contraction reduces over
// as the row index.  Two adjacent 16-row result tiles then hold, per lane,
// exactly eight reduction slots {4g..4g+3, 16+4g..16+4g+3} of a 32-wide
// contraction, and the probabilities feed the next contraction straight from
// registers; its other operand is read from LDS with the same slot order.
//
//   forward: S^T = K Q^T -> online softmax per query column -> O^T += V^T P^T
//   dq     : S^T, dP^T = V dO^T -> dS^T -> dQ^T += K^T dS^T
//   dk, dv : S = Q K^T, dP = dO V^T -> dV^T += dO^T P,  dK^T += Q^T dS
// The backward is two kernels (dq; dk and dv) so that every output element
// has exactly one writer: no atomics, bitwise deterministic.
#include "common.h"
#include "kernels.h"

namespace flglm {

namespace {

constexpr int kBlockN = 64;  // keys per tile (forward, dq)
constexpr int kThreads = 256;

struct SeqInfo {
  int r0, L, P;
};
__device__ __forceinline__ SeqInfo seq_info(const int32_t* cu, const int32_t* prefix, int s) {
  SeqInfo si;
  si.r0 = cu[s];
  si.L = cu[s + 1] - si.r0;
  si.P = prefix ? prefix[s] : 0;
  return si;
}
__device__ __forceinline__ bool visible(int i, int j, int L, int P) { return j < L && (j <= i || j < P); }

// Copy a ROWS x D tile (rows row0.. of a packed matrix, columns col0..) into
// LDS.  Row-major image: element (r, c) at S[r*D + swz(r, c/8)*8 + c%8].
// Transposed image: element (r, c) at S[c*ROWS + swz(c, r/8)*8 + r%8].
// Rows >= nrows are zero.  Work is spread over `nthr` threads starting at
// thread `t0`.
template <typename T, int ROWS, int D>
struct TileIO {
  static constexpr int NCH = ROWS * D / 8;           // 8-element chunks
  static constexpr int NBLK = (ROWS / 8) * (D / 8);  // 8x8 blocks
  __device__ static void rows(const T* G, long ld, int row0, int nrows, int col0, T* S, int t, int nthr) {
    for (int c = t; c < NCH; c += nthr) {
      const int r = c / (D / 8), ch = c % (D / 8);
      Vec8<T> v;
      if (r < nrows) v.load(G + (long)(row0 + r) * ld + col0 + ch * 8);
      else v.zero();
      v.store(S + r * D + swz(r, ch) * 8);
    }
  }
  // Loads 8x8 blocks and writes the row-major image (if Srow) and the
  // transposed image (if Scol).
  __device__ static void blocks(const T* G, long ld, int row0, int nrows, int col0, T* Srow, T* Scol, int t,
                                int nthr) {
    for (int b = t; b < NBLK; b += nthr) {
      const int rb = b % (ROWS / 8), cb = b / (ROWS / 8);
      Vec8<T> v[8], tr[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int r = rb * 8 + j;
        if (r < nrows) v[j].load(G + (long)(row0 + r) * ld + col0 + cb * 8);
        else v[j].zero();
      }
      if (Srow) {
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const int r = rb * 8 + j;
          v[j].store(Srow + r * D + swz(r, cb) * 8);
        }
      }
      if (Scol) {
        transpose8x8(v, tr);
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const int c = cb * 8 + j;
          tr[j].store(Scol + c * ROWS + swz(c, rb) * 8);
        }
      }
    }
  }
};

// Fragment of a row-major LDS image: row r, slots = columns 32*c + 8*g .. +7.
template <typename T, int D>
__device__ __forceinline__ frag_t<T> frag_rows(const T* S, int r, int c, int g) {
  Vec8<T> v;
  v.load(S + r * D + swz(r, 4 * c + g) * 8);
  return v.frag();
}
// Fragment of a transposed LDS image (row = contraction output index d, ROWS
// reduction columns): slots {32c + 4g .. +3, 32c + 16 + 4g .. +3}.
template <typename T, int ROWS>
__device__ __forceinline__ frag_t<T> frag_slots(const T* S, int d, int c, int g) {
  const int k1 = 32 * c + 4 * g, k2 = k1 + 16;
  Vec4<T> a, b;
  a.load(S + d * ROWS + swz(d, k1 >> 3) * 8 + (k1 & 7));
  b.load(S + d * ROWS + swz(d, k2 >> 3) * 8 + (k2 & 7));
  return join(a, b);
}

// Eight probabilities of two adjacent 16-row result tiles as one fragment.
template <typename T>
__device__ __forceinline__ frag_t<T> frag_pack(const float (&x)[4], const float (&y)[4]) {
  const float v[8] = {x[0], x[1], x[2], x[3], y[0], y[1], y[2], y[3]};
  return pack8(v, (T*)nullptr);
}

}  // namespace

// ---------------------------------------------------------------------------
// Forward.  Workgroup: 128 queries (4 waves x 2 subtiles of 16) of one
// (sequence, head); keys in tiles of 64, double-buffered in LDS.
// ---------------------------------------------------------------------------
template <typename T, int D>
__global__ void __launch_bounds__(kThreads) attn_fwd_kernel(AttnDesc a) {
  constexpr int QS = 2;
  constexpr int BM = 64 * QS;
  constexpr int NC = D / 32;
  __shared__ __attribute__((aligned(16))) T Ks[2][kBlockN * D];
  __shared__ __attribute__((aligned(16))) T Vt[2][D * kBlockN];

  const int s = blockIdx.z, h = blockIdx.y;
  const int qt = gridDim.x - 1 - blockIdx.x;  // longest-running (last) query tiles first
  const SeqInfo si = seq_info(a.cu_seqlens, a.prefix_len, s);
  const int q0 = qt * BM;
  if (q0 >= si.L) return;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int fr = lane & 15, fg = lane >> 4;
  const T* qkv = static_cast<const T*>(a.qkv);
  const long ld = a.ld_qkv;
  const int H = a.hidden;
  const float sl2 = kLog2e / sqrtf((float)D);

  frag_t<T> qf[QS][NC];
#pragma unroll
  for (int qs = 0; qs < QS; ++qs) {
    const int qi = q0 + 32 * w + 16 * qs + fr;
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      Vec8<T> v;
      if (qi < si.L) v.load(qkv + (long)(si.r0 + qi) * ld + h * D + 32 * c + 8 * fg);
      else v.zero();
      qf[qs][c] = v.frag();
    }
  }
  const int kv_end = min(si.L, max(q0 + BM, si.P));
  const int nkt = (kv_end + kBlockN - 1) / kBlockN;

  f32x4 acc[D / 16][QS];
#pragma unroll
  for (int dt = 0; dt < D / 16; ++dt)
#pragma unroll
    for (int qs = 0; qs < QS; ++qs) acc[dt][qs] = f32x4{0.f, 0.f, 0.f, 0.f};
  float m[QS], l[QS];
#pragma unroll
  for (int qs = 0; qs < QS; ++qs) { m[qs] = -INFINITY; l[qs] = 0.f; }

  auto load_tile = [&](int kt, int buf) {
    const int j0 = kt * kBlockN;
    const int n = min(kBlockN, si.L - j0);
    if (tid < 128)
      TileIO<T, kBlockN, D>::rows(qkv, ld, si.r0 + j0, n, H + h * D, Ks[buf], tid, 128);
    else
      TileIO<T, kBlockN, D>::blocks(qkv, ld, si.r0 + j0, n, 2 * H + h * D, nullptr, Vt[buf], tid - 128, 128);
  };

  load_tile(0, 0);
  __syncthreads();
  for (int kt = 0; kt < nkt; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < nkt) load_tile(kt + 1, buf ^ 1);
    const T* ks = Ks[buf];
    const T* vt = Vt[buf];
    const int j0 = kt * kBlockN;

    float p[QS][4][4];
#pragma unroll
    for (int qs = 0; qs < QS; ++qs) {
      f32x4 st[4];
#pragma unroll
      for (int at = 0; at < 4; ++at) {
        st[at] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int c = 0; c < NC; ++c) st[at] = mma16(frag_rows<T, D>(ks, 16 * at + fr, c, fg), qf[qs][c], st[at]);
      }
      const int qi = q0 + 32 * w + 16 * qs + fr;
      float mx = -INFINITY;
#pragma unroll
      for (int at = 0; at < 4; ++at)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int j = j0 + 16 * at + 4 * fg + i;
          const float v = visible(qi, j, si.L, si.P) ? st[at][i] * sl2 : -INFINITY;
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
      frag_t<T> pf[QS];
#pragma unroll
      for (int qs = 0; qs < QS; ++qs) pf[qs] = frag_pack<T>(p[qs][2 * c2], p[qs][2 * c2 + 1]);
#pragma unroll
      for (int dt = 0; dt < D / 16; ++dt) {
        const frag_t<T> vf = frag_slots<T, kBlockN>(vt, 16 * dt + fr, c2, fg);
#pragma unroll
        for (int qs = 0; qs < QS; ++qs) acc[dt][qs] = mma16(vf, pf[qs], acc[dt][qs]);
      }
    }
    __syncthreads();
  }

  T* o = static_cast<T*>(a.o);
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
      Vec4<T> ov;
      ov.set(v);
      ov.store(o + (long)(si.r0 + qi) * a.ld_o + h * D + 16 * dt + 4 * fg);
    }
    if (fg == 0) a.lse[(long)(si.r0 + qi) * a.num_heads + h] = m[qs] * 0.69314718055994531f + logf(lt);
  }
}

// ---------------------------------------------------------------------------
// Backward pre-pass: delta[t][h] = sum_d dO[t][h*D+d] * O[t][h*D+d].
// One wave per row.
// ---------------------------------------------------------------------------
template <typename T, int D>
__global__ void __launch_bounds__(256) attn_delta_kernel(const T* dout, long ld_do, const T* o, long ld_o,
                                                         float* delta, int T_, int H, int nh) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= T_) return;
  constexpr int CPH = D / 8;  // chunks per head
  const int nch = H / 8;
  for (int c0 = 0; c0 < nch; c0 += 64) {
    const int c = c0 + lane;
    float sacc = 0.f;
    if (c < nch) {
      Vec8<T> x, y;
      x.load(dout + (long)row * ld_do + c * 8);
      y.load(o + (long)row * ld_o + c * 8);
#pragma unroll
      for (int e = 0; e < 8; ++e) sacc += x.get(e) * y.get(e);
    }
#pragma unroll
    for (int off = CPH / 2; off > 0; off >>= 1) sacc += __shfl_xor(sacc, off, 64);
    if (c < nch && (lane % CPH) == 0) delta[(long)row * nh + c / CPH] = sacc;
  }
}

// Inverse rotation of a gradient held as lane tiles acc[dt] (rows d = 16dt +
// 4g + i): pairs (d, d + r/2) for d < r/2, angle -p*theta.
template <int D>
__device__ __forceinline__ void rope_bwd_tiles(f32x4 (&acc)[D / 16], int p, int r, int fg, const float* ct,
                                               const float* stb) {
  const int half = r / 2;
  const int ht = half / 16;
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
// Backward, dq.  Workgroup: 64 queries (4 waves x 16) of one (sequence,
// head); keys in tiles of 64 (K row-major and transposed, V row-major).
// ---------------------------------------------------------------------------
template <typename T, int D>
__global__ void __launch_bounds__(kThreads) attn_bwd_dq_kernel(AttnDesc a) {
  constexpr int BM = 64;
  constexpr int NC = D / 32;
  __shared__ __attribute__((aligned(16))) T Ks[kBlockN * D];
  __shared__ __attribute__((aligned(16))) T Kt[D * kBlockN];
  __shared__ __attribute__((aligned(16))) T Vs[kBlockN * D];

  const int s = blockIdx.z, h = blockIdx.y;
  const int qt = gridDim.x - 1 - blockIdx.x;
  const SeqInfo si = seq_info(a.cu_seqlens, a.prefix_len, s);
  const int q0 = qt * BM;
  if (q0 >= si.L) return;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int fr = lane & 15, fg = lane >> 4;
  const T* qkv = static_cast<const T*>(a.qkv);
  const T* dout = static_cast<const T*>(a.dout);
  const long ld = a.ld_qkv;
  const int H = a.hidden;
  const float sl2 = kLog2e / sqrtf((float)D);

  const int qi = q0 + 16 * w + fr;
  const bool qvalid = qi < si.L;
  frag_t<T> qf[NC], dof[NC];
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    Vec8<T> v, u;
    if (qvalid) {
      v.load(qkv + (long)(si.r0 + qi) * ld + h * D + 32 * c + 8 * fg);
      u.load(dout + (long)(si.r0 + qi) * a.ld_dout + h * D + 32 * c + 8 * fg);
    } else {
      v.zero();
      u.zero();
    }
    qf[c] = v.frag();
    dof[c] = u.frag();
  }
  const float lse2 = qvalid ? a.lse[(long)(si.r0 + qi) * a.num_heads + h] * kLog2e : 0.f;
  const float dlt = qvalid ? a.delta[(long)(si.r0 + qi) * a.num_heads + h] : 0.f;

  f32x4 acc[D / 16];
#pragma unroll
  for (int dt = 0; dt < D / 16; ++dt) acc[dt] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int kv_end = min(si.L, max(q0 + BM, si.P));
  const int nkt = (kv_end + kBlockN - 1) / kBlockN;
  for (int kt = 0; kt < nkt; ++kt) {
    const int j0 = kt * kBlockN;
    const int n = min(kBlockN, si.L - j0);
    __syncthreads();
    if (tid < 128)
      TileIO<T, kBlockN, D>::blocks(qkv, ld, si.r0 + j0, n, H + h * D, Ks, Kt, tid, 128);
    else
      TileIO<T, kBlockN, D>::rows(qkv, ld, si.r0 + j0, n, 2 * H + h * D, Vs, tid - 128, 128);
    __syncthreads();

    float ds[4][4];
#pragma unroll
    for (int at = 0; at < 4; ++at) {
      f32x4 st = f32x4{0.f, 0.f, 0.f, 0.f}, dp = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int c = 0; c < NC; ++c) {
        st = mma16(frag_rows<T, D>(Ks, 16 * at + fr, c, fg), qf[c], st);
        dp = mma16(frag_rows<T, D>(Vs, 16 * at + fr, c, fg), dof[c], dp);
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int j = j0 + 16 * at + 4 * fg + i;
        const float pr = (qvalid && visible(qi, j, si.L, si.P)) ? exp2f(st[i] * sl2 - lse2) : 0.f;
        ds[at][i] = pr * (dp[i] - dlt);
      }
    }
#pragma unroll
    for (int c2 = 0; c2 < 2; ++c2) {
      const frag_t<T> df = frag_pack<T>(ds[2 * c2], ds[2 * c2 + 1]);
#pragma unroll
      for (int dt = 0; dt < D / 16; ++dt) acc[dt] = mma16(frag_slots<T, kBlockN>(Kt, 16 * dt + fr, c2, fg), df, acc[dt]);
    }
  }
  if (!qvalid) return;
  const float sc = 1.f / sqrtf((float)D);
#pragma unroll
  for (int dt = 0; dt < D / 16; ++dt) acc[dt] *= sc;
  rope_bwd_tiles<D>(acc, qi, a.rotary_dim, fg, a.cos_t, a.sin_t);
  T* dq = static_cast<T*>(a.dqkv) + (long)(si.r0 + qi) * a.ld_dqkv + h * D;
#pragma unroll
  for (int dt = 0; dt < D / 16; ++dt) {
    const float v[4] = {acc[dt][0], acc[dt][1], acc[dt][2], acc[dt][3]};
    Vec4<T> ov;
    ov.set(v);
    ov.store(dq + 16 * dt + 4 * fg);
  }
}

// ---------------------------------------------------------------------------
// Backward, dk and dv.  Workgroup: 64 keys (4 waves x 16) of one (sequence,
// head); queries in tiles of 64 (Q and dO row-major and transposed).
// ---------------------------------------------------------------------------
template <typename T, int D>
__global__ void __launch_bounds__(kThreads) attn_bwd_dkdv_kernel(AttnDesc a) {
  constexpr int BK = 64;  // keys per workgroup
  constexpr int BQ = 64;  // queries per tile
  constexpr int NC = D / 32;
  __shared__ __attribute__((aligned(16))) T Qs[BQ * D];
  __shared__ __attribute__((aligned(16))) T Qt[D * BQ];
  __shared__ __attribute__((aligned(16))) T Os[BQ * D];
  __shared__ __attribute__((aligned(16))) T Ot[D * BQ];
  __shared__ float lse_s[BQ], dl_s[BQ];

  const int s = blockIdx.z, h = blockIdx.y;
  const int kt_ = gridDim.x - 1 - blockIdx.x;
  const SeqInfo si = seq_info(a.cu_seqlens, a.prefix_len, s);
  const int k0 = kt_ * BK;
  if (k0 >= si.L) return;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int fr = lane & 15, fg = lane >> 4;
  const T* qkv = static_cast<const T*>(a.qkv);
  const T* dout = static_cast<const T*>(a.dout);
  const long ld = a.ld_qkv;
  const int H = a.hidden;
  const float sl2 = kLog2e / sqrtf((float)D);

  const int kj = k0 + 16 * w + fr;
  const bool kvalid = kj < si.L;
  frag_t<T> kf[NC], vf[NC];
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    Vec8<T> v, u;
    if (kvalid) {
      v.load(qkv + (long)(si.r0 + kj) * ld + H + h * D + 32 * c + 8 * fg);
      u.load(qkv + (long)(si.r0 + kj) * ld + 2 * H + h * D + 32 * c + 8 * fg);
    } else {
      v.zero();
      u.zero();
    }
    kf[c] = v.frag();
    vf[c] = u.frag();
  }
  f32x4 dk[D / 16], dv[D / 16];
#pragma unroll
  for (int dt = 0; dt < D / 16; ++dt) { dk[dt] = f32x4{0.f, 0.f, 0.f, 0.f}; dv[dt] = dk[dt]; }

  const int q_start = (k0 < si.P) ? 0 : k0;
  for (int qb = (q_start / BQ) * BQ; qb < si.L; qb += BQ) {
    const int n = min(BQ, si.L - qb);
    __syncthreads();
    if (tid < 128)
      TileIO<T, BQ, D>::blocks(qkv, ld, si.r0 + qb, n, h * D, Qs, Qt, tid, 128);
    else
      TileIO<T, BQ, D>::blocks(dout, a.ld_dout, si.r0 + qb, n, h * D, Os, Ot, tid - 128, 128);
    if (tid < BQ) {
      const int q = qb + tid;
      lse_s[tid] = q < si.L ? a.lse[(long)(si.r0 + q) * a.num_heads + h] * kLog2e : 0.f;
      dl_s[tid] = q < si.L ? a.delta[(long)(si.r0 + q) * a.num_heads + h] : 0.f;
    }
    __syncthreads();

    float pr[4][4], ds[4][4];
#pragma unroll
    for (int qs = 0; qs < 4; ++qs) {
      f32x4 st = f32x4{0.f, 0.f, 0.f, 0.f}, dp = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int c = 0; c < NC; ++c) {
        st = mma16(frag_rows<T, D>(Qs, 16 * qs + fr, c, fg), kf[c], st);
        dp = mma16(frag_rows<T, D>(Os, 16 * qs + fr, c, fg), vf[c], dp);
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int ql = 16 * qs + 4 * fg + i;
        const int q = qb + ql;
        const float p = (kvalid && q < si.L && visible(q, kj, si.L, si.P)) ? exp2f(st[i] * sl2 - lse_s[ql]) : 0.f;
        pr[qs][i] = p;
        ds[qs][i] = p * (dp[i] - dl_s[ql]);
      }
    }
#pragma unroll
    for (int c2 = 0; c2 < 2; ++c2) {
      const frag_t<T> pf = frag_pack<T>(pr[2 * c2], pr[2 * c2 + 1]);
      const frag_t<T> df = frag_pack<T>(ds[2 * c2], ds[2 * c2 + 1]);
#pragma unroll
      for (int dt = 0; dt < D / 16; ++dt) {
        dv[dt] = mma16(frag_slots<T, BQ>(Ot, 16 * dt + fr, c2, fg), pf, dv[dt]);
        dk[dt] = mma16(frag_slots<T, BQ>(Qt, 16 * dt + fr, c2, fg), df, dk[dt]);
      }
    }
  }
  if (!kvalid) return;
  const float sc = 1.f / sqrtf((float)D);
#pragma unroll
  for (int dt = 0; dt < D / 16; ++dt) dk[dt] *= sc;
  rope_bwd_tiles<D>(dk, kj, a.rotary_dim, fg, a.cos_t, a.sin_t);
  T* row = static_cast<T*>(a.dqkv) + (long)(si.r0 + kj) * a.ld_dqkv + h * D;
#pragma unroll
  for (int dt = 0; dt < D / 16; ++dt) {
    const float vk[4] = {dk[dt][0], dk[dt][1], dk[dt][2], dk[dt][3]};
    const float vv[4] = {dv[dt][0], dv[dt][1], dv[dt][2], dv[dt][3]};
    Vec4<T> ok, ov;
    ok.set(vk);
    ov.set(vv);
    ok.store(row + H + 16 * dt + 4 * fg);
    ov.store(row + 2 * H + 16 * dt + 4 * fg);
  }
}

// ---------------------------------------------------------------------------
// Launchers
// ---------------------------------------------------------------------------
template <typename T, int D>
static hipError_t fwd_t(const AttnDesc& a, hipStream_t st) {
  dim3 grid((a.max_seqlen + 127) / 128, a.num_heads, a.num_seqs);
  hipLaunchKernelGGL((attn_fwd_kernel<T, D>), grid, dim3(kThreads), 0, st, a);
  return hipGetLastError();
}

template <typename T, int D>
static hipError_t delta_t(const AttnDesc& a, hipStream_t st) {
  hipLaunchKernelGGL((attn_delta_kernel<T, D>), dim3((a.total_tokens + 3) / 4), dim3(256), 0, st,
                     (const T*)a.dout, a.ld_dout, (const T*)a.o, a.ld_o, a.delta, a.total_tokens, a.hidden,
                     a.num_heads);
  return hipGetLastError();
}

hipError_t attn_delta(DType dt, const AttnDesc& a, hipStream_t st) {
  if (a.total_tokens <= 0) return hipSuccess;
  if (a.head_dim == 128) return dt == DT_BF16 ? delta_t<bf16, 128>(a, st) : delta_t<float, 128>(a, st);
  if (a.head_dim == 64) return dt == DT_BF16 ? delta_t<bf16, 64>(a, st) : delta_t<float, 64>(a, st);
  return hipErrorInvalidValue;
}

template <typename T, int D>
static hipError_t bwd_t(const AttnDesc& a, hipStream_t st) {
  hipError_t e = delta_t<T, D>(a, st);
  if (e != hipSuccess) return e;
  dim3 grid((a.max_seqlen + 63) / 64, a.num_heads, a.num_seqs);
  hipLaunchKernelGGL((attn_bwd_dkdv_kernel<T, D>), grid, dim3(kThreads), 0, st, a);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((attn_bwd_dq_kernel<T, D>), grid, dim3(kThreads), 0, st, a);
  return hipGetLastError();
}

// bf16 always runs on the LDS-DMA kernels (attention_bf16.hip), which take
// every supported shape, the P-tuning prefix included; these generic
// kernels serve the fp32 debug mode, which has no prefix.
hipError_t attn_fwd(DType dt, const AttnDesc& a, hipStream_t st) {
  if (a.num_seqs <= 0 || a.max_seqlen <= 0) return hipSuccess;
  if (dt == DT_BF16) return attn_bf16_ok(a) ? attn_fwd_bf16(a, st) : hipErrorInvalidValue;
  if (a.num_prefix > 0) return hipErrorInvalidValue;
  if (a.head_dim == 128) return fwd_t<float, 128>(a, st);
  if (a.head_dim == 64) return fwd_t<float, 64>(a, st);
  return hipErrorInvalidValue;
}

hipError_t attn_bwd(DType dt, const AttnDesc& a, hipStream_t st) {
  if (a.num_seqs <= 0 || a.max_seqlen <= 0) return hipSuccess;
  if (dt == DT_BF16) return attn_bf16_ok(a) ? attn_bwd_bf16(a, st) : hipErrorInvalidValue;
  if (a.num_prefix > 0) return hipErrorInvalidValue;
  if (a.head_dim == 128) return bwd_t<float, 128>(a, st);
  if (a.head_dim == 64) return bwd_t<float, 64>(a, st);
  return hipErrorInvalidValue;
}

}  // namespace flglm
