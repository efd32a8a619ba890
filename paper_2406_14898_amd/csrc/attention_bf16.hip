// bf16 attention over packed ragged sequences for gfx950 (the fp32 debug
// mode uses attention.hip).  Same contract as attention.hip: every
// workgroup stays inside one (sequence, head); key j is visible to query i
// iff j <= max(i, P - 1); scale 1/sqrt(d) (Appendix A: softmax(QK^T/sqrt(d_h))).
//
// Data movement:
//   * K, V (forward, dq) and Q, dO (dk/dv) tiles of 64 rows x d go from HBM
//     straight into LDS with buffer loads in LDS-DMA mode, double-buffered:
//     the next tile streams in while the current one is used.  Each tile
//     gets its own buffer resource, based at its first row and bounded at
//     the sequence end, so rows past it read as zero and offsets stay small
//     at any sequence length.
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
// Loops are unrolled over the two LDS slots so tile addresses are
// compile-time; per-lane fragment offsets are computed once; a wave skips
// key tiles it cannot see and masks only tiles that straddle the diagonal
// or the sequence end.
#include <type_traits>

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
// Query i of a sequence of L rows whose first P rows are its context sees
// keys j < L with j <= i or j < P: exactly the keys j < vis_end(i, L, P).
__device__ __forceinline__ int vis_end(int i, int L, int P) { return min(L, max(i + 1, P)); }
// Key j < L is seen by the queries i >= vis_start(j, P) (all of them when j
// is a context key); a key past the sequence end by none.
__device__ __forceinline__ int vis_start(int j, int L, int P) { return j >= L ? (1 << 30) : (j < P ? 0 : j); }

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

// Buffer resource over one 64-row tile of a sequence: rows row0 ..
// min(row0 + 64, L) - 1 of the rows starting at base (row stride ld
// elements); rows past the sequence end read as zero.  Rebasing per tile
// keeps every buffer offset below 64 rows, whatever the sequence length.
__device__ __forceinline__ i32x4 tile_rsrc(const bf16* base, long ld, int row0, int L) {
  return buf_rsrc(base + (long)row0 * ld, (uint32_t)((long)min(L - row0, kRows) * ld * 2));
}

// Per-lane element offsets of the fragment reads inside a [64][D] tile, so
// that every read in the loops is one base plus a compile-time offset:
//   row[c]: rows fr (+ 16 at), reduction slots 32c + 8g .. +7 (16-byte read);
//   tr[dt]: columns 16 dt + lane (two transpose reads over rows
//           {kb + 4g + e, kb + 16 + 4g + e}, e < 4; + kb D, + 16 D).
// Row offsets that are multiples of 8 leave the swizzle unchanged.
template <int D>
struct FragBase {
  int row[D / 32];
  int tr[D / 16];
  __device__ __forceinline__ void init(int fr, int fg) {
#pragma unroll
    for (int c = 0; c < D / 32; ++c) row[c] = fr * D + (((4 * c + fg) ^ swz<D>(fr)) << 3);
    const int r1 = 4 * fg + (fr >> 2);
#pragma unroll
    for (int dt = 0; dt < D / 16; ++dt) {
      const int col = 16 * dt + 4 * (fr & 3);
      tr[dt] = r1 * D + (((col >> 3) ^ swz<D>(r1)) << 3) + (col & 7);
    }
  }
};
__device__ __forceinline__ bf16x8 rd_row(const bf16* p) { return __builtin_bit_cast(bf16x8, ld16(p)); }
template <int D>
__device__ __forceinline__ bf16x8 rd_tr(const bf16* p) {
  i16x4 a = __builtin_amdgcn_ds_read_tr16_b64_v4i16((LDS_AS i16x4*)p);
  i16x4 b = __builtin_amdgcn_ds_read_tr16_b64_v4i16((LDS_AS i16x4*)(p + 16 * D));
  return __builtin_bit_cast(bf16x8, __builtin_shufflevector(a, b, 0, 1, 2, 3, 4, 5, 6, 7));
}

__device__ __forceinline__ bf16x8 pack_p(const f32x4& x, const f32x4& y) {
  return bf16x8{from_f32<bf16>(x[0]), from_f32<bf16>(x[1]), from_f32<bf16>(x[2]), from_f32<bf16>(x[3]),
                from_f32<bf16>(y[0]), from_f32<bf16>(y[1]), from_f32<bf16>(y[2]), from_f32<bf16>(y[3])};
}
__device__ __forceinline__ float ex2(float x) { return __builtin_amdgcn_exp2f(x); }  // exp2(-inf) = 0

// Sum over the 16 lanes of each row of the wave (lanes 16 g .. 16 g + 15) in
// a fixed order: an inclusive scan by DPP row shifts of 1, 2, 4 and 8, after
// which lane 16 g + 15 holds the row's sum.
__device__ __forceinline__ float row16_sum(float v) {
  v += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0x111, 0xf, 0xf, true));
  v += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0x112, 0xf, 0xf, true));
  v += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0x114, 0xf, 0xf, true));
  v += __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), 0x118, 0xf, 0xf, true));
  return v;
}

__device__ __forceinline__ void bar() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}
template <int V>
using Slot = std::integral_constant<int, V>;

// Inverse rotation of a gradient held as lane tiles acc[dt] (rows d = 16dt +
// 4g + i): pairs (d, d + r/2) for d < r/2, angle -p*theta.
template <int D, typename Acc>
__device__ __forceinline__ void rope_back(Acc& acc, int p, int r, int fg, const float* ct, const float* stb) {
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

// Workgroup -> (row tile, head, sequence), XCD-aware.  Workgroup i runs on
// XCD i % 8.  (sequence, head) groups are dealt round-robin to the XCDs
// (every XCD gets every eighth head of every sequence, which balances
// ragged lengths), and each group's row tiles run back to back on its XCD,
// so the tiles that stream the same K/V (or Q/dO) rows share one L2.  The
// tile order inside a group is reversed: the longest-running tiles start
// first.  Groups past the real count exit.
struct WgCoord {
  int tile, h, s;
};
__device__ __forceinline__ WgCoord wg_coord(int ntiles, int nh) {
  const int i = blockIdx.x, x = i % 8, j = i / 8;
  const int gi = j / ntiles;
  WgCoord c;
  c.tile = ntiles - 1 - (j - gi * ntiles);
  const int g = gi * 8 + x;
  c.h = g % nh;
  c.s = g / nh;
  return c;
}
__host__ __forceinline__ dim3 wg_grid(int ntiles, int nh, int nseq) {
  const long groups = ((long)nh * nseq + 7) / 8 * 8;
  return dim3((unsigned)(groups * ntiles));
}

// The block's P-tuning v2 prefix for head h: n rows in ntiles key tiles;
// buffer resources over [n, hidden] bf16 keys / values starting at column
// h * D (rows past n read as zero).
struct PrefixKV {
  int n, ntiles;
  i32x4 rk, rv;
  __device__ __forceinline__ PrefixKV(const AttnDesc& a, int h, int D) {
    n = a.num_prefix;
    ntiles = (n + kRows - 1) / kRows;
    const uint32_t bytes = n > 0 ? (uint32_t)(((long)n * a.hidden - (long)h * D) * 2) : 0u;
    rk = buf_rsrc(static_cast<const bf16*>(a.pk) + h * D, bytes);
    rv = buf_rsrc(static_cast<const bf16*>(a.pv) + h * D, bytes);
  }
};

// Key tile [j0, j0 + 64) against queries [qlo, qlo + nq): none visible / all
// visible (keys inside the sequence, each at or before every query or in the
// prefix).  Wave-uniform, so only diagonal and ragged tiles pay for masking.
__device__ __forceinline__ bool tile_dark(int j0, int qlo, int nq, int P) { return j0 > qlo + nq - 1 && j0 >= P; }
__device__ __forceinline__ bool tile_full(int j0, int qlo, int L, int P) {
  return j0 + kRows <= L && (j0 + kRows - 1 <= qlo || j0 + kRows <= P);
}

// Stored softmax gradient (dS, bf16) of the backward, in 64 x 64 tiles, one
// per (query tile, key tile) pair that holds a visible pair: query tile qt of
// a sequence meets the ntp prefix key tiles and the sequence's key tiles
// kt < max(qt + 1, np), np = ceil(P / 64) (the context keys every query
// sees).  Tiles of a sequence and head are numbered row by row: query tile
// qt starts at ds_row_off(qt) and its key tiles follow in order, prefix
// first.  A tile holds dS^T in the order the dk/dv kernel's lanes hold it:
// 16-byte chunk c = (2 w + p) 64 + 16 g + r holds, for key 16 w + r, the
// queries 32 p + 4 g + e (e < 4) and 32 p + 16 + 4 g + e - 4 (e >= 4), so
// every store is a whole 1 KB block; keys 32 c2 .. + 31 are the contiguous
// half c2.
__host__ __device__ __forceinline__ long ds_row_off(int qt, int ntp, int np) {
  if (qt <= np) return (long)qt * (ntp + np);
  return (long)np * (ntp + np) + (long)(qt - np) * ntp + ((long)qt * (qt + 1) - (long)np * (np + 1)) / 2;
}
__host__ __device__ __forceinline__ long ds_seq_tiles(int L, int P, int ntp) {
  return ds_row_off((L + kRows - 1) / kRows, ntp, (P + kRows - 1) / kRows);
}
constexpr long kDsTileElems = (long)kRows * kRows;

// ---------------------------------------------------------------------------
// Forward: 128 queries per workgroup (4 waves x 32), key tiles of 64.
// ---------------------------------------------------------------------------
template <int D>
__global__ void __launch_bounds__(256, 2) fwd_kernel(AttnDesc a) {
  constexpr int NC = D / 32, ND = D / 16, QS = 2, BM = 128;
  __shared__ __attribute__((aligned(1024))) bf16 Ks[2][kRows * D];
  __shared__ __attribute__((aligned(1024))) bf16 Vs[2][kRows * D];

  const WgCoord wc = wg_coord((a.max_seqlen + BM - 1) / BM, a.num_heads);
  if (wc.s >= a.num_seqs) return;
  const int s = wc.s, h = wc.h, q0 = wc.tile * BM;
  const SeqB si = seqb(a.cu_seqlens, a.prefix_len, s);
  if (q0 >= si.L) return;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int fr = lane & 15, fg = lane >> 4;
  const bf16* qkv = static_cast<const bf16*>(a.qkv);
  const long ld = a.ld_qkv;
  const int H = a.hidden;
  const float sl2 = kLog2e / sqrtf((float)D);
  FragBase<D> fb;
  fb.init(fr, fg);

  const bf16* kbase = qkv + (long)si.r0 * ld + H + h * D;
  const bf16* vbase = kbase + H;
  // key tiles 0 .. ntp-1: the prefix (row stride H), then the sequence's own
  const PrefixKV px(a, h, D);
  const int kv_end = min(si.L, max(q0 + BM, si.P));
  const int nkt = px.ntiles + (kv_end + kRows - 1) / kRows;
  const uint32_t lds_k = FL_LDS_ADDR(&Ks[0][0]), lds_v = FL_LDS_ADDR(&Vs[0][0]);
  auto issue = [&](int kt) {
    const uint32_t sk = lds_k + (kt & 1) * (kRows * D * 2), sv = lds_v + (kt & 1) * (kRows * D * 2);
    if (kt < px.ntiles) {
      dma_tile<D>(px.rk, H, kt * kRows, sk, w, lane);
      dma_tile<D>(px.rv, H, kt * kRows, sv, w, lane);
    } else {
      const int j0 = (kt - px.ntiles) * kRows;
      dma_tile<D>(tile_rsrc(kbase, ld, j0, si.L), ld, 0, sk, w, lane);
      dma_tile<D>(tile_rsrc(vbase, ld, j0, si.L), ld, 0, sv, w, lane);
    }
  };
  issue(0);

  const int qlo = q0 + 32 * w;  // this wave's queries: qlo + 16 qs + fr
  bf16x8 qf[QS][NC];
#pragma unroll
  for (int qs = 0; qs < QS; ++qs) {
    const int qi = qlo + 16 * qs + fr;
#pragma unroll
    for (int c = 0; c < NC; ++c)
      qf[qs][c] = qi < si.L ? __builtin_bit_cast(bf16x8, ld16(qkv + (long)(si.r0 + qi) * ld + h * D + 32 * c + 8 * fg))
                            : bf16x8{};
  }
#pragma unroll
  for (int qs = 0; qs < QS; ++qs)
#pragma unroll
    for (int c = 0; c < NC; ++c) settle(qf[qs][c]);
  f32x4 acc[ND][QS];
#pragma unroll
  for (int dt = 0; dt < ND; ++dt)
#pragma unroll
    for (int qs = 0; qs < QS; ++qs) acc[dt][qs] = f32x4{0.f, 0.f, 0.f, 0.f};
  // running maximum (log2 units of the scaled scores) and sum; key 0 is
  // visible to every query, so the maximum is finite after the first tile
  float m[QS], l[QS];
#pragma unroll
  for (int qs = 0; qs < QS; ++qs) { m[qs] = -INFINITY; l[qs] = 0.f; }

  auto step = [&](auto slot, int kt) {
    constexpr int SL = decltype(slot)::value;
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    bar();  // tile kt landed for every wave; the other slot is free
    if (kt + 1 < nkt) issue(kt + 1);
    const bool pre = kt < px.ntiles;
    const int j0 = (pre ? kt : kt - px.ntiles) * kRows;
    if (!pre && tile_dark(j0, qlo, 32, si.P)) return;
    const bool full = pre ? j0 + kRows <= px.n : tile_full(j0, qlo, si.L, si.P);
    const bf16* ks = Ks[SL];
    const bf16* vs = Vs[SL];
    f32x4 st[QS][4];
#pragma unroll
    for (int qs = 0; qs < QS; ++qs)
#pragma unroll
      for (int at = 0; at < 4; ++at) st[qs][at] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      bf16x8 kf[4];
#pragma unroll
      for (int at = 0; at < 4; ++at) kf[at] = rd_row(ks + 16 * at * D + fb.row[c]);
#pragma unroll
      for (int qs = 0; qs < QS; ++qs)
#pragma unroll
        for (int at = 0; at < 4; ++at) st[qs][at] = mma16(kf[at], qf[qs][c], st[qs][at]);
    }
#pragma unroll
    for (int qs = 0; qs < QS; ++qs) {
      if (!full) {
        // key j0 + 16 at + 4 fg + i is visible iff 16 at + i < rel
        const int rel = (pre ? px.n : vis_end(qlo + 16 * qs + fr, si.L, si.P)) - j0 - 4 * fg;
#pragma unroll
        for (int at = 0; at < 4; ++at)
#pragma unroll
          for (int i = 0; i < 4; ++i) st[qs][at][i] = 16 * at + i < rel ? st[qs][at][i] : -INFINITY;
      }
      float mx = st[qs][0][0];
#pragma unroll
      for (int at = 0; at < 4; ++at)
#pragma unroll
        for (int i = 0; i < 4; ++i) mx = fmaxf(mx, st[qs][at][i]);
      mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
      mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
      const float mnew = fmaxf(m[qs], mx * sl2);
      const float alpha = ex2(m[qs] - mnew);
      m[qs] = mnew;
      float ls = 0.f;
#pragma unroll
      for (int at = 0; at < 4; ++at)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float e = ex2(fmaf(st[qs][at][i], sl2, -mnew));
          st[qs][at][i] = e;
          ls += e;
        }
      l[qs] = l[qs] * alpha + ls;
      if (__builtin_amdgcn_ballot_w64(alpha != 1.f)) {
#pragma unroll
        for (int dt = 0; dt < ND; ++dt) acc[dt][qs] *= alpha;
      }
    }
#pragma unroll
    for (int c2 = 0; c2 < 2; ++c2) {
      bf16x8 pf[QS];
#pragma unroll
      for (int qs = 0; qs < QS; ++qs) pf[qs] = pack_p(st[qs][2 * c2], st[qs][2 * c2 + 1]);
#pragma unroll
      for (int dt = 0; dt < ND; ++dt) {
        const bf16x8 vf = rd_tr<D>(vs + 32 * c2 * D + fb.tr[dt]);
#pragma unroll
        for (int qs = 0; qs < QS; ++qs) acc[dt][qs] = mma16(vf, pf[qs], acc[dt][qs]);
      }
    }
  };
  for (int kt = 0; kt < nkt; kt += 2) {
    step(Slot<0>{}, kt);
    if (kt + 1 < nkt) step(Slot<1>{}, kt + 1);
  }

  bf16* o = static_cast<bf16*>(a.o);
#pragma unroll
  for (int qs = 0; qs < QS; ++qs) {
    float lt = l[qs];
    lt += __shfl_xor(lt, 16, 64);
    lt += __shfl_xor(lt, 32, 64);
    const int qi = qlo + 16 * qs + fr;
    if (qi >= si.L) continue;
    const float inv = 1.f / lt;
#pragma unroll
    for (int dt = 0; dt < ND; ++dt) {
      const float v[4] = {acc[dt][qs][0] * inv, acc[dt][qs][1] * inv, acc[dt][qs][2] * inv, acc[dt][qs][3] * inv};
      Vec4<bf16> ov;
      ov.set(v);
      ov.store(o + (long)(si.r0 + qi) * a.ld_o + h * D + 16 * dt + 4 * fg);
    }
    if (fg == 0) a.lse[(long)(si.r0 + qi) * a.num_heads + h] = m[qs] * 0.69314718055994531f + logf(lt);
  }
}

// ---------------------------------------------------------------------------
// Backward, dq: 128 queries per workgroup (4 waves x 32), key tiles of 64.
// Rows past the sequence end read as zero, so they add nothing to dq; only
// the causal / prefix mask needs applying, on diagonal tiles.
// ---------------------------------------------------------------------------
template <int D>
__global__ void __launch_bounds__(256, 2) dq_kernel(AttnDesc a) {
  constexpr int NC = D / 32, ND = D / 16, QS = 2, BM = 128;
  __shared__ __attribute__((aligned(1024))) bf16 Ks[2][kRows * D];
  __shared__ __attribute__((aligned(1024))) bf16 Vs[2][kRows * D];

  const WgCoord wc = wg_coord((a.max_seqlen + BM - 1) / BM, a.num_heads);
  if (wc.s >= a.num_seqs) return;
  const int s = wc.s, h = wc.h, q0 = wc.tile * BM;
  const SeqB si = seqb(a.cu_seqlens, a.prefix_len, s);
  if (q0 >= si.L) return;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int fr = lane & 15, fg = lane >> 4;
  const bf16* qkv = static_cast<const bf16*>(a.qkv);
  const bf16* dout = static_cast<const bf16*>(a.dout);
  const long ld = a.ld_qkv;
  const int H = a.hidden;
  const float sl2 = kLog2e / sqrtf((float)D);
  FragBase<D> fb;
  fb.init(fr, fg);

  const bf16* kbase = qkv + (long)si.r0 * ld + H + h * D;
  const bf16* vbase = kbase + H;
  const PrefixKV px(a, h, D);
  const int kv_end = min(si.L, max(q0 + BM, si.P));
  const int nkt = px.ntiles + (kv_end + kRows - 1) / kRows;
  const uint32_t lds_k = FL_LDS_ADDR(&Ks[0][0]), lds_v = FL_LDS_ADDR(&Vs[0][0]);
  auto issue = [&](int kt) {
    const uint32_t sk = lds_k + (kt & 1) * (kRows * D * 2), sv = lds_v + (kt & 1) * (kRows * D * 2);
    if (kt < px.ntiles) {
      dma_tile<D>(px.rk, H, kt * kRows, sk, w, lane);
      dma_tile<D>(px.rv, H, kt * kRows, sv, w, lane);
    } else {
      const int j0 = (kt - px.ntiles) * kRows;
      dma_tile<D>(tile_rsrc(kbase, ld, j0, si.L), ld, 0, sk, w, lane);
      dma_tile<D>(tile_rsrc(vbase, ld, j0, si.L), ld, 0, sv, w, lane);
    }
  };
  issue(0);

  const int qlo = q0 + 32 * w;
  bf16x8 qf[QS][NC], dof[QS][NC];
  float lse2[QS], dlt[QS];
#pragma unroll
  for (int qs = 0; qs < QS; ++qs) {
    const int qi = qlo + 16 * qs + fr;
    const bool ok = qi < si.L;
    const long r = si.r0 + qi;
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      qf[qs][c] = ok ? __builtin_bit_cast(bf16x8, ld16(qkv + r * ld + h * D + 32 * c + 8 * fg)) : bf16x8{};
      dof[qs][c] = ok ? __builtin_bit_cast(bf16x8, ld16(dout + r * a.ld_dout + h * D + 32 * c + 8 * fg)) : bf16x8{};
    }
    lse2[qs] = ok ? a.lse[r * a.num_heads + h] * kLog2e : 0.f;
    dlt[qs] = ok ? a.delta[r * a.num_heads + h] : 0.f;
  }
#pragma unroll
  for (int qs = 0; qs < QS; ++qs) {
#pragma unroll
    for (int c = 0; c < NC; ++c) { settle(qf[qs][c]); settle(dof[qs][c]); }
    settle(lse2[qs]);
    settle(dlt[qs]);
  }
  f32x4 acc[ND][QS];
#pragma unroll
  for (int dt = 0; dt < ND; ++dt)
#pragma unroll
    for (int qs = 0; qs < QS; ++qs) acc[dt][qs] = f32x4{0.f, 0.f, 0.f, 0.f};

  auto step = [&](auto slot, int kt) {
    constexpr int SL = decltype(slot)::value;
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    bar();
    if (kt + 1 < nkt) issue(kt + 1);
    const bool pre = kt < px.ntiles;
    const int j0 = (pre ? kt : kt - px.ntiles) * kRows;
    if (!pre && tile_dark(j0, qlo, 32, si.P)) return;
    const bool full = pre ? j0 + kRows <= px.n : tile_full(j0, qlo, si.L, si.P);
    const bf16* ks = Ks[SL];
    const bf16* vs = Vs[SL];
    // keys in two halves of 32 (reduction half c2 of the dq product), which
    // keeps half of the score and dP tiles live at a time
#pragma unroll
    for (int c2 = 0; c2 < 2; ++c2) {
      f32x4 st[QS][2], dp[QS][2];
#pragma unroll
      for (int qs = 0; qs < QS; ++qs)
#pragma unroll
        for (int u = 0; u < 2; ++u) { st[qs][u] = f32x4{0.f, 0.f, 0.f, 0.f}; dp[qs][u] = st[qs][u]; }
#pragma unroll
      for (int c = 0; c < NC; ++c) {
#pragma unroll
        for (int u = 0; u < 2; ++u) {
          const int at = 2 * c2 + u;
          const bf16x8 kf = rd_row(ks + 16 * at * D + fb.row[c]);
          const bf16x8 vf = rd_row(vs + 16 * at * D + fb.row[c]);
#pragma unroll
          for (int qs = 0; qs < QS; ++qs) {
            st[qs][u] = mma16(kf, qf[qs][c], st[qs][u]);
            dp[qs][u] = mma16(vf, dof[qs][c], dp[qs][u]);
          }
        }
      }
      bf16x8 df[QS];
#pragma unroll
      for (int qs = 0; qs < QS; ++qs) {
        const int qi = qlo + 16 * qs + fr;
#pragma unroll
        for (int u = 0; u < 2; ++u)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const float pr = ex2(fmaf(st[qs][u][i], sl2, -lse2[qs]));
            st[qs][u][i] = pr * (dp[qs][u][i] - dlt[qs]);
          }
        // masking only where the tile straddles the diagonal, the prefix end
        // or the sequence end (a wave-uniform test: full tiles skip it)
        if (!full) {
          // key j0 + 32 c2 + 16 u + 4 fg + i is visible iff 16 u + i < rel
          const int rel = (pre ? px.n : vis_end(qi, si.L, si.P)) - j0 - 32 * c2 - 4 * fg;
#pragma unroll
          for (int u = 0; u < 2; ++u)
#pragma unroll
            for (int i = 0; i < 4; ++i) st[qs][u][i] = 16 * u + i < rel ? st[qs][u][i] : 0.f;
        }
        df[qs] = pack_p(st[qs][0], st[qs][1]);
      }
#pragma unroll
      for (int dt = 0; dt < ND; ++dt) {
        const bf16x8 kt_ = rd_tr<D>(ks + 32 * c2 * D + fb.tr[dt]);
#pragma unroll
        for (int qs = 0; qs < QS; ++qs) acc[dt][qs] = mma16(kt_, df[qs], acc[dt][qs]);
      }
    }
  };
  for (int kt = 0; kt < nkt; kt += 2) {
    step(Slot<0>{}, kt);
    if (kt + 1 < nkt) step(Slot<1>{}, kt + 1);
  }

  const float sc = 1.f / sqrtf((float)D);
#pragma unroll
  for (int qs = 0; qs < QS; ++qs) {
    const int qi = qlo + 16 * qs + fr;
    if (qi >= si.L) continue;
    f32x4 g[ND];
#pragma unroll
    for (int dt = 0; dt < ND; ++dt) g[dt] = acc[dt][qs] * sc;
    rope_back<D>(g, qi, a.rotary_dim, fg, a.cos_t, a.sin_t);
    bf16* dq = static_cast<bf16*>(a.dqkv) + (long)(si.r0 + qi) * a.ld_dqkv + h * D;
#pragma unroll
    for (int dt = 0; dt < ND; ++dt) {
      const float v[4] = {g[dt][0], g[dt][1], g[dt][2], g[dt][3]};
      Vec4<bf16> ov;
      ov.set(v);
      ov.store(dq + 16 * dt + 4 * fg);
    }
  }
}

// ---------------------------------------------------------------------------
// Backward, dk and dv: 64 keys per workgroup (4 waves x 16), query tiles of
// 64 with their LSE and delta rows.  Query rows past the sequence end read
// as zero (and their LSE and delta as zero), which makes their dS and their
// dO rows zero: they add nothing, so again only diagonal tiles are masked.
// ---------------------------------------------------------------------------
// DS: also store dS^T (the tiles dq_ds_kernel reads; see ds_row_off).
template <int D, bool DS>
__global__ void __launch_bounds__(256, 2) dkdv_kernel(AttnDesc a) {
  constexpr int NC = D / 32, ND = D / 16, BK = 64;
  __shared__ __attribute__((aligned(1024))) bf16 Qs[2][kRows * D];
  __shared__ __attribute__((aligned(1024))) bf16 Os[2][kRows * D];
  __shared__ __attribute__((aligned(256))) float Ls[2][kRows];
  __shared__ __attribute__((aligned(256))) float Ds[2][kRows];

  // Key tiles in work order u = 0, 1, ...: the prefix tiles (every query of
  // the sequence sees them), then the sequence's own from row 0 (the tile at
  // row k0 meets the queries from k0 on), i.e. longest-running first.
  const int ntp = (a.num_prefix + BK - 1) / BK, nts = (a.max_seqlen + BK - 1) / BK;
  const WgCoord wc = wg_coord(ntp + nts, a.num_heads);
  if (wc.s >= a.num_seqs) return;
  const int u = ntp + nts - 1 - wc.tile;
  const bool pre = u < ntp;
  const int s = wc.s, h = wc.h, k0 = (pre ? u : u - ntp) * BK;
  const SeqB si = seqb(a.cu_seqlens, a.prefix_len, s);
  if (!pre && k0 >= si.L) return;
  // the bias-sum row of this tile, read now rather than at the epilogue
  const int bias_row = (DS && a.bias_part && !pre) ? a.tile_base[s] + k0 / kRows : 0;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int fr = lane & 15, fg = lane >> 4;
  const bf16* qkv = static_cast<const bf16*>(a.qkv);
  const bf16* dout = static_cast<const bf16*>(a.dout);
  const long ld = a.ld_qkv;
  const int H = a.hidden, nh = a.num_heads;
  const float sl2 = kLog2e / sqrtf((float)D);
  FragBase<D> fb;
  fb.init(fr, fg);

  const bf16* qbase = qkv + (long)si.r0 * ld + h * D;
  const bf16* obase = dout + (long)si.r0 * a.ld_dout + h * D;
  const float* lbase = a.lse + (long)si.r0 * nh + h;
  const float* dbase = a.delta + (long)si.r0 * nh + h;
  const int qstart = (pre || k0 < si.P) ? 0 : k0 / kRows;
  const int nqt = (si.L + kRows - 1) / kRows;
  const uint32_t lds_q = FL_LDS_ADDR(&Qs[0][0]), lds_o = FL_LDS_ADDR(&Os[0][0]);
  const uint32_t lds_l = FL_LDS_ADDR(&Ls[0][0]), lds_d = FL_LDS_ADDR(&Ds[0][0]);
  // query tile qt lives in slot (qt - qstart) & 1
  auto issue = [&](int qt) {
    const int slot = (qt - qstart) & 1, q0 = qt * kRows;
    dma_tile<D>(tile_rsrc(qbase, ld, q0, si.L), ld, 0, lds_q + slot * (kRows * D * 2), w, lane);
    dma_tile<D>(tile_rsrc(obase, a.ld_dout, q0, si.L), a.ld_dout, 0, lds_o + slot * (kRows * D * 2), w, lane);
    // LSE (scaled on use) and delta rows: 64 x 4 bytes each
    const uint32_t voff = (uint32_t)(lane * nh) * 4u;
    const uint32_t nb = (uint32_t)(min(si.L - q0, kRows) * nh * 4 - h * 4);
    if (w == 0) dma_lds<4>(buf_rsrc(lbase + (long)q0 * nh, nb), lds_l + slot * (kRows * 4), voff);
    if (w == 1) dma_lds<4>(buf_rsrc(dbase + (long)q0 * nh, nb), lds_d + slot * (kRows * 4), voff);
  };
  issue(qstart);

  const int klo = k0 + 16 * w;  // this wave's keys: klo + fr (prefix rows for a prefix tile)
  const int kj = klo + fr;
  const bool kvalid = kj < (pre ? a.num_prefix : si.L);
  const int kstart = pre ? 0 : vis_start(kj, si.L, si.P);
  // key / value rows of this lane: the prefix buffers (row stride H) or qkv
  const bf16* krow = pre ? static_cast<const bf16*>(a.pk) + (long)kj * H + h * D
                         : qkv + (long)(si.r0 + kj) * ld + H + h * D;
  const bf16* vrow = pre ? static_cast<const bf16*>(a.pv) + (long)kj * H + h * D
                         : qkv + (long)(si.r0 + kj) * ld + 2 * H + h * D;
  bf16x8 kf[NC], vf[NC];
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    kf[c] = kvalid ? __builtin_bit_cast(bf16x8, ld16(krow + 32 * c + 8 * fg)) : bf16x8{};
    vf[c] = kvalid ? __builtin_bit_cast(bf16x8, ld16(vrow + 32 * c + 8 * fg)) : bf16x8{};
  }
#pragma unroll
  for (int c = 0; c < NC; ++c) { settle(kf[c]); settle(vf[c]); }
  f32x4 dk[ND], dv[ND];
#pragma unroll
  for (int dt = 0; dt < ND; ++dt) { dk[dt] = f32x4{0.f, 0.f, 0.f, 0.f}; dv[dt] = dk[dt]; }
  // stored dS^T: this lane's chunks of the tile of query tile qt (tile
  // column u of its tile row)
  bf16* ds_seq = nullptr;
  int ds_np = 0;
  if constexpr (DS) {
    ds_np = (si.P + kRows - 1) / kRows;
    ds_seq = static_cast<bf16*>(a.ds) + (a.ds_off[s] + (long)h * ds_seq_tiles(si.L, si.P, ntp)) * kDsTileElems +
             (2 * w * 64 + lane) * 8;
  }
  // two 1 KB stores per wave and query tile (chunk pairs p = 0, 1), the same
  // number on every step
  auto ds_store = [&](int qt, int p, u32x4 v) {
    // streamed (non-temporal): dS is read once, by the dq kernel, and must not
    // evict the Q / dO tiles the other workgroups of this head re-read
    __builtin_nontemporal_store(
        v, reinterpret_cast<u32x4*>(ds_seq + (ds_row_off(qt, ntp, ds_np) + u) * kDsTileElems + p * 64 * 8));
  };

  auto step = [&](auto slot, int qt) {
    constexpr int SL = decltype(slot)::value;
    // The next tile's DMA was issued before this wave's dS stores of the
    // previous step (two): waiting for all but those two is enough.
    if (DS && qt != qstart)
      asm volatile("s_waitcnt vmcnt(2)" ::: "memory");
    else
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    bar();
    if (qt + 1 < nqt) issue(qt + 1);
    const int qb = qt * kRows;
    // queries [qb, qb + 64) against keys [klo, klo + 16); prefix keys are
    // visible to all
    if (!pre && qb + kRows - 1 < klo && klo >= si.P) {
      if constexpr (DS) {
        ds_store(qt, 0, u32x4{0u, 0u, 0u, 0u});
        ds_store(qt, 1, u32x4{0u, 0u, 0u, 0u});
      }
      return;
    }
    const bool full = pre || qb >= klo + 15 || klo + 15 < si.P;
    const bf16* qs_ = Qs[SL];
    const bf16* os_ = Os[SL];
    const float* ls_ = Ls[SL];
    const float* dls = Ds[SL];
    // Software pipeline with a fixed issue order (scheduling barriers):
    //   phase 1, steps n = (qs, c): S^T and dP^T tiles, fragment reads two
    //   steps ahead; the softmax-gradient arithmetic of query group qs - 1
    //   runs between the matrix instructions of group qs;
    //   phase 3, steps n = (c2, dt): dV^T and dK^T, transpose reads two steps
    //   ahead.
    constexpr int N1 = 4 * NC, N3 = 2 * ND;
    f32x4 st[4], dp[4], pr[4], dsv[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) { st[q] = f32x4{0.f, 0.f, 0.f, 0.f}; dp[q] = st[q]; }
    f32x4 lq[2], dq[2];
    bf16x8 pf[2], df[2];
    auto rd1 = [&](int n, bf16x8& x, bf16x8& y) {
      const int q = n / NC, c = n % NC;
      x = rd_row(qs_ + 16 * q * D + fb.row[c]);
      y = rd_row(os_ + 16 * q * D + fb.row[c]);
    };
    auto elem = [&](int q) {
      // rows qb + 16 q + 4 g + i of this lane's column kj
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float pv = ex2(fmaf(st[q][i], sl2, -lq[q & 1][i] * kLog2e));
        pr[q][i] = pv;
        dsv[q][i] = pv * (dp[q][i] - dq[q & 1][i]);
      }
      if (!full) {  // diagonal or ragged tiles only (wave-uniform)
        // query qb + 16 q + 4 fg + i sees this lane's key iff 16 q + i >= rel
        const int rel = kstart - qb - 4 * fg;
#pragma unroll
        for (int i = 0; i < 4; ++i)
          if (16 * q + i < rel) { pr[q][i] = 0.f; dsv[q][i] = 0.f; }
      }
      if (q & 1) {
        pf[q >> 1] = pack_p(pr[q - 1], pr[q]);
        df[q >> 1] = pack_p(dsv[q - 1], dsv[q]);
        if constexpr (DS)  // a key past the sequence end stores zeros (its dS is not masked)
          ds_store(qt, q >> 1, kvalid ? __builtin_bit_cast(u32x4, df[q >> 1]) : u32x4{0u, 0u, 0u, 0u});
      }
    };
    bf16x8 fq[3], fo[3];
    rd1(0, fq[0], fo[0]);
    rd1(1, fq[1], fo[1]);
#pragma unroll
    for (int n = 0; n < N1; ++n) {
      const int q = n / NC, c = n % NC;
      if (n + 2 < N1) rd1(n + 2, fq[(n + 2) % 3], fo[(n + 2) % 3]);
      if (c == 0) {
        lq[q & 1] = __builtin_bit_cast(f32x4, ld16(ls_ + 16 * q + 4 * fg));
        dq[q & 1] = __builtin_bit_cast(f32x4, ld16(dls + 16 * q + 4 * fg));
      }
      __builtin_amdgcn_sched_barrier(0);
      st[q] = mma16(fq[n % 3], kf[c], st[q]);
      dp[q] = mma16(fo[n % 3], vf[c], dp[q]);
      __builtin_amdgcn_sched_barrier(0);
      if (c == 1 && q >= 1) elem(q - 1);
    }
    auto rd3 = [&](int n, bf16x8& x, bf16x8& y) {
      const int c2 = n / ND, dt = n % ND;
      x = rd_tr<D>(os_ + 32 * c2 * D + fb.tr[dt]);
      y = rd_tr<D>(qs_ + 32 * c2 * D + fb.tr[dt]);
    };
    bf16x8 to[3], tq[3];
    rd3(0, to[0], tq[0]);
    elem(3);
    rd3(1, to[1], tq[1]);
#pragma unroll
    for (int n = 0; n < N3; ++n) {
      const int c2 = n / ND, dt = n % ND;
      if (n + 2 < N3) rd3(n + 2, to[(n + 2) % 3], tq[(n + 2) % 3]);
      __builtin_amdgcn_sched_barrier(0);
      dv[dt] = mma16(to[n % 3], pf[c2], dv[dt]);
      dk[dt] = mma16(tq[n % 3], df[c2], dk[dt]);
      __builtin_amdgcn_sched_barrier(0);
    }
  };
  for (int qt = qstart; qt < nqt; qt += 2) {
    step(Slot<0>{}, qt);
    if (qt + 1 < nqt) step(Slot<1>{}, qt + 1);
  }
  const float sc = 1.f / sqrtf((float)D);
#pragma unroll
  for (int dt = 0; dt < ND; ++dt) dk[dt] *= sc;
  if (pre) {
    if (!kvalid) return;
    // this sequence's share of the prefix gradients, fp32, unrotated
    float* pk_out = a.dprefix_part + ((long)s * a.num_prefix + kj) * H + h * D;
    float* pv_out = pk_out + (long)a.num_seqs * a.num_prefix * H;
#pragma unroll
    for (int dt = 0; dt < ND; ++dt) {
      st16(pk_out + 16 * dt + 4 * fg, __builtin_bit_cast(u32x4, dk[dt]));
      st16(pv_out + 16 * dt + 4 * fg, __builtin_bit_cast(u32x4, dv[dt]));
    }
    return;
  }
  if (kvalid) rope_back<D>(dk, kj, a.rotary_dim, fg, a.cos_t, a.sin_t);
  Vec4<bf16> ok[ND], ov[ND];
#pragma unroll
  for (int dt = 0; dt < ND; ++dt) {
    const float vk[4] = {dk[dt][0], dk[dt][1], dk[dt][2], dk[dt][3]};
    const float vv[4] = {dv[dt][0], dv[dt][1], dv[dt][2], dv[dt][3]};
    ok[dt].set(vk);
    ov[dt].set(vv);
  }
  if constexpr (DS) {
    if (a.bias_part) {
      // column sums of the stored dk and dv rows of this 64-key tile: over
      // the wave's 16 keys (row16_sum), then the four waves in order
      // through the (now free) Q tile
      float* red = reinterpret_cast<float*>(&Qs[0][0]);  // [wave][dk | dv][D]
      __syncthreads();  // every wave is past its last reads of the tiles
#pragma unroll
      for (int dt = 0; dt < ND; ++dt) {
        f32x4 sk, sv;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          sk[e] = row16_sum(kvalid ? ok[dt].get(e) : 0.f);
          sv[e] = row16_sum(kvalid ? ov[dt].get(e) : 0.f);
        }
        if (fr == 15) {
          st16(red + (w * 2 + 0) * D + 16 * dt + 4 * fg, __builtin_bit_cast(u32x4, sk));
          st16(red + (w * 2 + 1) * D + 16 * dt + 4 * fg, __builtin_bit_cast(u32x4, sv));
        }
      }
      __syncthreads();
      for (int c = tid; c < 2 * D; c += 256) {
        const float t = ((red[c] + red[2 * D + c]) + red[4 * D + c]) + red[6 * D + c];
        a.bias_part[(long)bias_row * 3 * H + (c < D ? H : 2 * H) + h * D + c % D] = t;
      }
    }
  }
  if (!kvalid) return;
  bf16* row = static_cast<bf16*>(a.dqkv) + (long)(si.r0 + kj) * a.ld_dqkv + h * D;
#pragma unroll
  for (int dt = 0; dt < ND; ++dt) {
    ok[dt].store(row + H + 16 * dt + 4 * fg);
    ov[dt].store(row + 2 * H + 16 * dt + 4 * fg);
  }
}

// ---------------------------------------------------------------------------
// Backward, dq from the stored dS: dq = scale sum_k dS[q][k] K[k] (no
// recomputation of S and dP).  256 queries per workgroup, one 64-row query
// tile per wave, key tiles in halves of 32 through three LDS stages: per
// stage, the half K tile and the matching halves of the four dS^T tiles of
// the workgroup's query tiles come in by DMA (a tile that does not exist,
// i.e. holds no visible pair, reads as zero), and both operands are read
// with transpose reads.  The workgroup walks the key tiles its last query
// tile sees; a wave whose own query tile does not see a key tile skips it.
// ---------------------------------------------------------------------------
// dS^T chunk c of a tile sits at LDS chunk c ^ (4 ((c >> 4) & 3)): the
// transpose reads (16 lanes: 4 keys x 4 query groups) then hit 16 distinct
// bank groups.
__device__ __forceinline__ int ds_swz(int c) { return c ^ (((c >> 4) & 3) << 2); }

template <int D>
__global__ void __launch_bounds__(256, 2) dq_ds_kernel(AttnDesc a) {
  constexpr int ND = D / 16, QS = 4, BM = 256, NS = 3, HR = 32;  // stages, rows per half tile
  constexpr int KCH = D / 8;                                      // 16-byte chunks per K row
  constexpr int KDMA = HR * KCH / 64 / 4;                         // K DMA instructions per wave per stage
  constexpr int DMA = KDMA + 4;                                   // + one per dS half tile
  constexpr int HALF = HR * kRows;                                // elements of a dS half tile
  __shared__ __attribute__((aligned(1024))) bf16 Ks[NS][HR * D];
  __shared__ __attribute__((aligned(1024))) bf16 Ss[NS][4][HALF];

  const WgCoord wc = wg_coord((a.max_seqlen + BM - 1) / BM, a.num_heads);
  if (wc.s >= a.num_seqs) return;
  const int s = wc.s, h = wc.h, q0 = wc.tile * BM;
  const SeqB si = seqb(a.cu_seqlens, a.prefix_len, s);
  if (q0 >= si.L) return;
  // the bias-sum row of this workgroup's first query tile, read now rather
  // than at the epilogue
  const int bias_row0 = a.bias_part ? a.tile_base[s] + q0 / kRows : 0;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int fr = lane & 15, fg = lane >> 4;
  const bf16* qkv = static_cast<const bf16*>(a.qkv);
  const long ld = a.ld_qkv;
  const int H = a.hidden;
  FragBase<D> fb;
  fb.init(fr, fg);
  // dS fragment of query group qs: keys 4 fg + (s / 4) (+ 16) of the half,
  // queries 16 qs + 4 (s % 4) .. + 3, s = fr; byte offset of the first read
  // for qs = 0 (+ 1 KB per query pair, + 8 bytes for an odd group, + 2 KB
  // for the second read)
  const int t4 = fr & 3;
  const uint32_t ds_rd = (uint32_t)((t4 * 16 + ((4 * fg + (fr >> 2)) ^ (4 * t4))) * 16);

  const bf16* kbase = qkv + (long)si.r0 * ld + H + h * D;
  const PrefixKV px(a, h, D);
  const int ntp = px.ntiles, np = (si.P + kRows - 1) / kRows, nt = (si.L + kRows - 1) / kRows;
  const int qt0 = q0 / kRows, qlast = min(qt0 + 3, nt - 1);
  const int nkt = ntp + max(qlast + 1, np);  // key tiles of the last query tile
  const int nst = 2 * nkt;                   // stages: (key tile, half)
  const int qt = qt0 + w;                    // this wave's query tile
  const int my_nkt = qt < nt ? ntp + max(qt + 1, np) : 0;
  const bf16* ds_seq =
      static_cast<const bf16*>(a.ds) + (a.ds_off[s] + (long)h * ds_seq_tiles(si.L, si.P, ntp)) * kDsTileElems;
  const uint32_t lds_k = FL_LDS_ADDR(&Ks[0][0]), lds_s = FL_LDS_ADDR(&Ss[0][0][0]);
  // per-lane source offsets: K rows (as dma_tile), dS chunk of this lane
  const uint32_t ds_src = (uint32_t)(ds_swz(w * 64 + lane) * 16);
  auto issue = [&](int g) {
    const int kc = g >> 1, c2 = g & 1, slot = g % NS;
    const uint32_t sk = lds_k + slot * (HR * D * 2);
    // a half past the sequence end (row0 >= L) gets no records: reads zero
    const int row0 = (kc - ntp) * kRows + HR * c2;
    i32x4 rk = kc < ntp ? px.rk
                        : buf_rsrc(kbase + (long)row0 * ld, (uint32_t)((long)max(0, min(si.L - row0, HR)) * ld * 2));
    rk = i32x4{__builtin_amdgcn_readfirstlane(rk[0]), __builtin_amdgcn_readfirstlane(rk[1]),
               __builtin_amdgcn_readfirstlane(rk[2]), __builtin_amdgcn_readfirstlane(rk[3])};
    const int r0 = kc < ntp ? kc * kRows + HR * c2 : 0;
    const long ldk = kc < ntp ? H : ld;
#pragma unroll
    for (int i = 0; i < KDMA; ++i) {
      const int inst = i * 4 + w;
      const int row = inst * (64 / KCH) + lane / KCH;
      const int q = (lane % KCH) ^ swz<D>(row);
      dma_lds<16>(rk, sk + inst * 1024, (uint32_t)((long)(r0 + row) * ldk + q * 8) * 2u);
    }
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const int q = qt0 + t;
      const bool has = q < nt && kc < ntp + max(q + 1, np);
      const bf16* src = ds_seq + (has ? (ds_row_off(q, ntp, np) + kc) * kDsTileElems + c2 * HALF : 0);
      dma_lds<16>(buf_rsrc(src, has ? (uint32_t)(HALF * 2) : 0u),
                  lds_s + (slot * 4 + t) * (uint32_t)(HALF * 2) + w * 1024, ds_src);
    }
  };
  issue(0);
  if (nst > 1) issue(1);

  f32x4 acc[ND][QS];
#pragma unroll
  for (int dt = 0; dt < ND; ++dt)
#pragma unroll
    for (int qs = 0; qs < QS; ++qs) acc[dt][qs] = f32x4{0.f, 0.f, 0.f, 0.f};

  for (int g = 0; g < nst; ++g) {
    // stage g landed (stage g + 1, if issued, may still be in flight)
    if (g + 1 < nst)
      asm volatile("s_waitcnt vmcnt(%0)" ::"n"(DMA) : "memory");
    else
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    bar();  // and every wave is past stage g - 1, whose slot stage g + 2 takes
    if (g + 2 < nst) issue(g + 2);
    if ((g >> 1) >= my_nkt) continue;
    // query groups (16 rows) of this wave that no key of the half sees (on
    // its diagonal tile) or past the sequence end: their dS is zero
    const int kc = g >> 1, kh = (kc - ntp) * kRows + HR * (g & 1);
    auto idle = [&](int qs) {
      const int q16 = qt * kRows + 16 * qs;
      return (kc >= ntp && q16 + 15 < kh && kh >= si.P) || q16 >= si.L;
    };
    const int slot = g % NS;
    const bf16* ks = Ks[slot];
    const char* ss = reinterpret_cast<const char*>(Ss[slot][w]);
    bf16x8 df[QS];
#pragma unroll
    for (int qs = 0; qs < QS; ++qs) {
      const char* p = ss + ds_rd + (qs >> 1) * 1024 + (qs & 1) * 8;
      i16x4 x = __builtin_amdgcn_ds_read_tr16_b64_v4i16((LDS_AS i16x4*)(p));
      i16x4 y = __builtin_amdgcn_ds_read_tr16_b64_v4i16((LDS_AS i16x4*)(p + 2048));
      df[qs] = __builtin_bit_cast(bf16x8, __builtin_shufflevector(x, y, 0, 1, 2, 3, 4, 5, 6, 7));
    }
    bf16x8 kt_[ND];
#pragma unroll
    for (int dt = 0; dt < ND; ++dt) kt_[dt] = rd_tr<D>(ks + fb.tr[dt]);
#pragma unroll
    for (int qs = 0; qs < QS; ++qs) {
      if (idle(qs)) continue;
#pragma unroll
      for (int dt = 0; dt < ND; ++dt) acc[dt][qs] = mma16(kt_[dt], df[qs], acc[dt][qs]);
    }
  }

  const float sc = 1.f / sqrtf((float)D);
  // column sums of the stored dq rows of this wave's query tile: this
  // lane's rows in query-group order, then over the 16 lanes (row16_sum)
  f32x4 bsum[ND];
#pragma unroll
  for (int dt = 0; dt < ND; ++dt) bsum[dt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int qs = 0; qs < QS; ++qs) {
    const int qi = qt * kRows + 16 * qs + fr;
    if (qi >= si.L) continue;
    f32x4 g[ND];
#pragma unroll
    for (int dt = 0; dt < ND; ++dt) g[dt] = acc[dt][qs] * sc;
    rope_back<D>(g, qi, a.rotary_dim, fg, a.cos_t, a.sin_t);
    bf16* dq = static_cast<bf16*>(a.dqkv) + (long)(si.r0 + qi) * a.ld_dqkv + h * D;
#pragma unroll
    for (int dt = 0; dt < ND; ++dt) {
      const float v[4] = {g[dt][0], g[dt][1], g[dt][2], g[dt][3]};
      Vec4<bf16> ov;
      ov.set(v);
      ov.store(dq + 16 * dt + 4 * fg);
#pragma unroll
      for (int e = 0; e < 4; ++e) bsum[dt][e] += ov.get(e);
    }
  }
  if (a.bias_part && qt < nt) {
    // over the wave's 16 lanes of a column (row16_sum): lane 16 g + 15 holds
    // columns 16 dt + 4 g .. + 3 of the whole 64-row tile
    float* out = a.bias_part + (long)(bias_row0 + w) * 3 * H + h * D;
#pragma unroll
    for (int dt = 0; dt < ND; ++dt) {
      f32x4 t;
#pragma unroll
      for (int e = 0; e < 4; ++e) t[e] = row16_sum(bsum[dt][e]);
      if (fr == 15) st16(out + 16 * dt + 4 * fg, __builtin_bit_cast(u32x4, t));
    }
  }
}

// Tile offsets of the stored dS: off[s] = sum over sequences before s of
// num_heads * ds_seq_tiles, off[S] = the total (one workgroup, chunked scan).
// With tile_base: tile_base[s] = the 64-row tiles of the sequences before s.
__global__ void __launch_bounds__(256) ds_offsets_kernel(const int32_t* cu, const int32_t* prefix, int S, int nh,
                                                         int ntp, int64_t* off, int32_t* tile_base) {
  __shared__ long sh[2][256];
  const int t = threadIdx.x;
  long carry = 0, carry_t = 0;
  for (int s0 = 0; s0 < S; s0 += 256) {
    const int s = s0 + t;
    long v = 0, vt = 0;
    if (s < S) {
      const int L = cu[s + 1] - cu[s];
      v = (long)nh * ds_seq_tiles(L, prefix ? prefix[s] : 0, ntp);
      vt = (L + kRows - 1) / kRows;
    }
    sh[0][t] = v;
    sh[1][t] = vt;
    __syncthreads();
    for (int o = 1; o < 256; o <<= 1) {
      const long x = t >= o ? sh[0][t - o] : 0, xt = t >= o ? sh[1][t - o] : 0;
      __syncthreads();
      sh[0][t] += x;
      sh[1][t] += xt;
      __syncthreads();
    }
    if (s < S) {
      off[s] = carry + sh[0][t] - v;
      if (tile_base) tile_base[s] = (int32_t)(carry_t + sh[1][t] - vt);
    }
    carry += sh[0][255];
    carry_t += sh[1][255];
    __syncthreads();
  }
  if (t == 0) {
    off[S] = carry;
    if (tile_base) tile_base[S] = (int32_t)carry_t;
  }
}

template <int D>
hipError_t fwd_launch(const AttnDesc& a, hipStream_t st) {
  const dim3 grid = wg_grid((a.max_seqlen + 127) / 128, a.num_heads, a.num_seqs);
  hipLaunchKernelGGL((fwd_kernel<D>), grid, dim3(256), 0, st, a);
  return hipGetLastError();
}

template <int D>
hipError_t bwd_launch(const AttnDesc& a, hipStream_t st) {
  hipError_t e = attn_delta(DT_BF16, a, st);
  if (e != hipSuccess) return e;
  const dim3 gkv = wg_grid((a.num_prefix + 63) / 64 + (a.max_seqlen + 63) / 64, a.num_heads, a.num_seqs);
  if (a.ds) {
    // dk, dv and the stored dS, then dq from dS
    if ((e = attn_ds_offsets(a, st)) != hipSuccess) return e;
    hipLaunchKernelGGL((dkdv_kernel<D, true>), gkv, dim3(256), 0, st, a);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    const dim3 gq = wg_grid((a.max_seqlen + 255) / 256, a.num_heads, a.num_seqs);
    hipLaunchKernelGGL((dq_ds_kernel<D>), gq, dim3(256), 0, st, a);
    return hipGetLastError();
  }
  hipLaunchKernelGGL((dkdv_kernel<D, false>), gkv, dim3(256), 0, st, a);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  const dim3 gq = wg_grid((a.max_seqlen + 127) / 128, a.num_heads, a.num_seqs);
  hipLaunchKernelGGL((dq_kernel<D>), gq, dim3(256), 0, st, a);
  return hipGetLastError();
}

}  // namespace

hipError_t attn_ds_offsets(const AttnDesc& a, hipStream_t st) {
  hipLaunchKernelGGL(ds_offsets_kernel, dim3(1), dim3(256), 0, st, a.cu_seqlens, a.prefix_len, a.num_seqs,
                     a.num_heads, (a.num_prefix + kRows - 1) / kRows, a.ds_off, a.bias_part ? a.tile_base : nullptr);
  return hipGetLastError();
}

// Buffer resources are rebased per 64-row tile, so any sequence length
// works; head dims 64 and 128.
bool attn_bf16_ok(const AttnDesc& a) { return a.head_dim == 64 || a.head_dim == 128; }

hipError_t attn_fwd_bf16(const AttnDesc& a, hipStream_t st) {
  if (a.num_seqs <= 0 || a.max_seqlen <= 0) return hipSuccess;
  return a.head_dim == 128 ? fwd_launch<128>(a, st) : fwd_launch<64>(a, st);
}

size_t attn_ds_tiles(const int32_t* cu, const int32_t* prefix, int num_seqs, int num_heads, int num_prefix) {
  const int ntp = (num_prefix + kRows - 1) / kRows;
  size_t n = 0;
  for (int s = 0; s < num_seqs; ++s) n += (size_t)num_heads * ds_seq_tiles(cu[s + 1] - cu[s], prefix ? prefix[s] : 0, ntp);
  return n;
}

hipError_t attn_bwd_bf16(const AttnDesc& a, hipStream_t st) {
  if (a.num_seqs <= 0 || a.max_seqlen <= 0) return hipSuccess;
  return a.head_dim == 128 ? bwd_launch<128>(a, st) : bwd_launch<64>(a, st);
}

}  // namespace flglm
