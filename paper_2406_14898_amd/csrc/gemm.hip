// Matrix-core GEMM for every linear layer of the block, forward and backward.
//
//   C[m, n] (op)= sum_k A(m, k) * B(n, k)
//
// Each operand is either "K-contiguous" (element (r, k) at P[r * ld + k]) or
// "MN-contiguous" (element (r, k) at P[k * ld + r]).  The three uses:
//   forward   y  = x W^T        A = x  (K-contig)   B = W  (K-contig)
//   dgrad     dx = dy W         A = dy (K-contig)   B = W  (MN-contig)
//   wgrad     dW += dy^T x      A = dy (MN-contig)  B = x  (MN-contig)
// MN-contiguous tiles are transposed in registers (8x8 blocks) on their way
// into LDS, so the LDS image of both operands is always K-contiguous and the
// inner loop is the same for all three.
//
// Tiling: a workgroup computes a BM x BN tile with BK = 64 reduction steps,
// double-buffered in LDS with a one-tile register prefetch.  Each wave owns
// a (16*WTM) x (16*WTN) sub-tile built from 16x16 matrix-core tiles.  The
// matrix-core tile is issued as D[n][m] (B rows first) so that a lane ends
// up with four consecutive output columns of one row, which the epilogue
// stores as one 8- or 16-byte vector.
#include <algorithm>

#include "common.h"
#include "kernels.h"

namespace flglm {


struct GemmArgs {
  const void* A;
  const void* B;
  void* C;
  int M, N, K;
  long lda, ldb, ldc;
  const void* bias;
  const void* R;
  long ldr;
  void* C2;
  long ldc2;
  const void* Z;
  long ldz;
  int nb;  // rows of B that exist (see GemmDesc::b_rows)
  float res_scale;
};

__device__ __forceinline__ float gelu_f(float z) {
  const float c = 0.7978845608028654f, a = 0.044715f;
  return 0.5f * z * (1.f + tanhf(c * (z + a * z * z * z)));
}
__device__ __forceinline__ float gelu_grad_f(float z) {
  const float c = 0.7978845608028654f, a = 0.044715f;
  float t = tanhf(c * (z + a * z * z * z));
  return 0.5f * (1.f + t) + 0.5f * z * (1.f - t * t) * c * (1.f + 3.f * a * z * z);
}

// Logical tile id for workgroup `wg`: workgroups are dealt round-robin to the
// 8 XCDs, so consecutive logical ids are regrouped onto one XCD (sharing its
// L2), then mapped to (tile_m, tile_n) in groups of GROUP_M tile rows.
__device__ __forceinline__ void tile_coords(int wg, int nwg, int tiles_m, int tiles_n, int& tm, int& tn) {
  constexpr int kXcd = 8;
  constexpr int kGroupM = 8;
  int q = nwg / kXcd, r = nwg % kXcd;
  int x = wg % kXcd, j = wg / kXcd;
  int id = (x < r) ? x * (q + 1) + j : r * (q + 1) + (x - r) * q + j;
  int per_group = kGroupM * tiles_n;
  int group = id / per_group;
  int first_m = group * kGroupM;
  int gsize = min(tiles_m - first_m, kGroupM);
  int in_group = id % per_group;
  tm = first_m + in_group % gsize;
  tn = in_group / gsize;
}

template <typename T, int BM, int BN, int WTM, int WTN, bool AK, bool BK_, int EPI>
struct GemmCfg {
  static constexpr int BK = 64;
  static constexpr int NWM = BM / (16 * WTM);
  static constexpr int NWN = BN / (16 * WTN);
  static constexpr int NT = 64 * NWM * NWN;
};

// Loads one ROWS x 64 operand tile (rows r0.., reduction k0..) into registers.
template <typename T, int ROWS, int NT, bool KCONTIG>
struct TileLoader;

template <typename T, int ROWS, int NT>
struct TileLoader<T, ROWS, NT, true> {
  static constexpr int CPT = ROWS * 8 / NT;  // 8-element chunks per thread
  static_assert(CPT * NT == ROWS * 8, "tile/threads mismatch");
  Vec8<T> v[CPT];
  __device__ __forceinline__ void load(const T* P, long ld, int r0, int rlim, int k0, int tid) {
#pragma unroll
    for (int i = 0; i < CPT; ++i) {
      int c = tid + i * NT;
      int row = c >> 3, kc = c & 7;
      if (r0 + row < rlim) v[i].load(P + (long)(r0 + row) * ld + k0 + kc * 8);
      else v[i].zero();
    }
  }
  __device__ __forceinline__ void store(T* S, int tid) const {
#pragma unroll
    for (int i = 0; i < CPT; ++i) {
      int c = tid + i * NT;
      int row = c >> 3, kc = c & 7;
      v[i].store(S + row * 64 + swz(row, kc) * 8);
    }
  }
};

template <typename T, int ROWS, int NT>
struct TileLoader<T, ROWS, NT, false> {
  static constexpr int NBLK = (ROWS / 8) * 8;  // 8x8 blocks per tile
  static constexpr int BPT = (NBLK + NT - 1) / NT;
  static_assert(NBLK % NT == 0 || NBLK < NT, "tile/threads mismatch");
  Vec8<T> v[BPT][8];
  __device__ __forceinline__ void load(const T* P, long ld, int r0, int rlim, int k0, int klim, int tid) {
#pragma unroll
    for (int b = 0; b < BPT; ++b) {
      int blk = tid + b * NT;
      if (blk >= NBLK) break;
      int rb = blk % (ROWS / 8), kb = blk / (ROWS / 8);
      int row = r0 + rb * 8;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        int k = k0 + kb * 8 + j;
        if (k < klim && row < rlim) v[b][j].load(P + (long)k * ld + row);
        else v[b][j].zero();
      }
    }
  }
  __device__ __forceinline__ void store(T* S, int tid) const {
#pragma unroll
    for (int b = 0; b < BPT; ++b) {
      int blk = tid + b * NT;
      if (blk >= NBLK) break;
      int rb = blk % (ROWS / 8), kb = blk / (ROWS / 8);
      Vec8<T> t[8];
      transpose8x8(v[b], t);
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        int row = rb * 8 + j;
        t[j].store(S + row * 64 + swz(row, kb) * 8);
      }
    }
  }
};

template <typename T, int BM, int BN, int WTM, int WTN, bool AK, bool BKc, int EPI>
__global__ void __launch_bounds__(64 * (BM / (16 * WTM)) * (BN / (16 * WTN)))
gemm_kernel(GemmArgs p) {
  using Cfg = GemmCfg<T, BM, BN, WTM, WTN, AK, BKc, EPI>;
  constexpr int NT = Cfg::NT;
  constexpr int BK = 64;
  __shared__ __attribute__((aligned(16))) T As[2][BM * BK];
  __shared__ __attribute__((aligned(16))) T Bs[2][BN * BK];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave % Cfg::NWM, wn = wave / Cfg::NWM;
  const int tiles_m = (p.M + BM - 1) / BM, tiles_n = p.N / BN;
  int tm, tn;
  tile_coords(blockIdx.x, gridDim.x, tiles_m, tiles_n, tm, tn);
  const int m0 = tm * BM, n0 = tn * BN;

  const T* A = static_cast<const T*>(p.A);
  const T* B = static_cast<const T*>(p.B);

  TileLoader<T, BM, NT, AK> la;
  TileLoader<T, BN, NT, BKc> lb;
  auto load_tiles = [&](int k0) {
    if constexpr (AK) la.load(A, p.lda, m0, p.M, k0, tid);
    else la.load(A, p.lda, m0, p.M, k0, p.K, tid);
    if constexpr (BKc) lb.load(B, p.ldb, n0, p.nb, k0, tid);
    else lb.load(B, p.ldb, n0, p.N, k0, p.nb, tid);
  };

  f32x4 acc[WTN][WTM];
#pragma unroll
  for (int i = 0; i < WTN; ++i)
#pragma unroll
    for (int j = 0; j < WTM; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  const int nk = (p.K + BK - 1) / BK;
  load_tiles(0);
  la.store(As[0], tid);
  lb.store(Bs[0], tid);
  __syncthreads();

  const int fr = lane & 15, fg = lane >> 4;
  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < nk) load_tiles((kt + 1) * BK);
    const T* as = As[buf];
    const T* bs = Bs[buf];
#pragma unroll
    for (int kk = 0; kk < BK / 32; ++kk) {
      const int ch = kk * 4 + fg;
      frag_t<T> af[WTM], bfr[WTN];
#pragma unroll
      for (int j = 0; j < WTM; ++j) {
        int row = wm * 16 * WTM + 16 * j + fr;
        Vec8<T> t;
        t.load(as + row * BK + swz(row, ch) * 8);
        af[j] = t.frag();
      }
#pragma unroll
      for (int i = 0; i < WTN; ++i) {
        int row = wn * 16 * WTN + 16 * i + fr;
        Vec8<T> t;
        t.load(bs + row * BK + swz(row, ch) * 8);
        bfr[i] = t.frag();
      }
#pragma unroll
      for (int i = 0; i < WTN; ++i)
#pragma unroll
        for (int j = 0; j < WTM; ++j) acc[i][j] = mma16(bfr[i], af[j], acc[i][j]);
    }
    if (kt + 1 < nk) {
      la.store(As[buf ^ 1], tid);
      lb.store(Bs[buf ^ 1], tid);
    }
    __syncthreads();
  }

  // Epilogue: lane holds C[m][n .. n+3].
#pragma unroll
  for (int j = 0; j < WTM; ++j) {
    const int m = m0 + wm * 16 * WTM + 16 * j + fr;
    if (m >= p.M) continue;
#pragma unroll
    for (int i = 0; i < WTN; ++i) {
      const int n = n0 + wn * 16 * WTN + 16 * i + 4 * fg;
      float v[4] = {acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3]};
      if constexpr (EPI == EPI_ACC_F32) {
        float* C = static_cast<float*>(p.C) + (long)m * p.ldc + n;
        Vec4<float> c;
        c.load(C);
        float o[4] = {c.get(0) + v[0], c.get(1) + v[1], c.get(2) + v[2], c.get(3) + v[3]};
        c.set(o);
        c.store(C);
      } else {
        if constexpr (EPI == EPI_BIAS || EPI == EPI_BIAS_RES || EPI == EPI_BIAS_GELU) {
          Vec4<T> b;
          b.load(static_cast<const T*>(p.bias) + n);
#pragma unroll
          for (int r = 0; r < 4; ++r) v[r] += b.get(r);
        }
        if constexpr (EPI == EPI_BIAS_RES || EPI == EPI_RES) {
          Vec4<T> rr;
          rr.load(static_cast<const T*>(p.R) + (long)m * p.ldr + n);
#pragma unroll
          for (int r = 0; r < 4; ++r) v[r] += p.res_scale * rr.get(r);
        }
        if constexpr (EPI == EPI_GELU_BWD) {
          Vec4<T> z;
          z.load(static_cast<const T*>(p.Z) + (long)m * p.ldz + n);
#pragma unroll
          for (int r = 0; r < 4; ++r) v[r] *= gelu_grad_f(z.get(r));
        }
        Vec4<T> o;
        o.set(v);
        if (EPI != EPI_BIAS_GELU || p.C) o.store(static_cast<T*>(p.C) + (long)m * p.ldc + n);
        if constexpr (EPI == EPI_BIAS_GELU) {
          float g[4];
#pragma unroll
          for (int r = 0; r < 4; ++r) g[r] = gelu_f(v[r]);
          Vec4<T> og;
          og.set(g);
          og.store(static_cast<T*>(p.C2) + (long)m * p.ldc2 + n);
        }
      }
    }
  }
}

// ---------------------------------------------------------------------------
// Launchers
// ---------------------------------------------------------------------------

template <typename T, int BM, int BN, int WTM, int WTN, bool AK, bool BKc, int EPI>
static hipError_t launch_cfg(const GemmArgs& a, hipStream_t st) {
  using Cfg = GemmCfg<T, BM, BN, WTM, WTN, AK, BKc, EPI>;
  int tiles = ((a.M + BM - 1) / BM) * (a.N / BN);
  if (tiles == 0) return hipSuccess;
  hipLaunchKernelGGL((gemm_kernel<T, BM, BN, WTM, WTN, AK, BKc, EPI>), dim3(tiles), dim3(Cfg::NT), 0, st, a);
  return hipGetLastError();
}

template <typename T, bool AK, bool BKc, int EPI>
static hipError_t launch_layout(const GemmArgs& a, hipStream_t st) {
  if constexpr (sizeof(T) == 2) {
    if (a.N % 256 == 0) return launch_cfg<T, 256, 256, 8, 8, AK, BKc, EPI>(a, st);
    return launch_cfg<T, 256, 128, 8, 4, AK, BKc, EPI>(a, st);
  } else {
    if (a.N % 128 == 0) return launch_cfg<T, 128, 128, 4, 4, AK, BKc, EPI>(a, st);
    return launch_cfg<T, 128, 64, 4, 2, AK, BKc, EPI>(a, st);
  }
}

template <typename T, GemmLayout L>
static hipError_t dispatch_layout(int epi, const GemmArgs& a, hipStream_t st) {
  if constexpr (L == GEMM_NT) {
    switch (epi) {
      case EPI_STORE: return launch_layout<T, true, true, EPI_STORE>(a, st);
      case EPI_BIAS: return launch_layout<T, true, true, EPI_BIAS>(a, st);
      case EPI_BIAS_RES: return launch_layout<T, true, true, EPI_BIAS_RES>(a, st);
      case EPI_BIAS_GELU: return launch_layout<T, true, true, EPI_BIAS_GELU>(a, st);
    }
  } else if constexpr (L == GEMM_NN) {
    switch (epi) {
      case EPI_STORE: return launch_layout<T, true, false, EPI_STORE>(a, st);
      case EPI_GELU_BWD: return launch_layout<T, true, false, EPI_GELU_BWD>(a, st);
      case EPI_RES: return launch_layout<T, true, false, EPI_RES>(a, st);
    }
  } else {
    if (epi == EPI_ACC_F32) return launch_layout<T, false, false, EPI_ACC_F32>(a, st);
  }
  return hipErrorInvalidValue;
}

hipError_t gemm(DType dt, GemmLayout layout, int epi, const GemmDesc& d, hipStream_t st) {
  if (dt == DT_BF16 && gemm_bf16_dma_ok(layout, d)) return gemm_bf16_dma(layout, epi, d, st);
  // A weight-gradient GEMM whose operands span 2^31 bytes or more along the
  // reduction (many tokens times a wide row) is cut along the reduction into
  // pieces the DMA kernel can address; its epilogue accumulates, so the
  // pieces add up in order.
  if (dt == DT_BF16 && layout == GEMM_TN && epi == EPI_ACC_F32 && d.K > 64) {
    const long ld = d.lda > d.ldb ? d.lda : d.ldb;
    const long kc = ((1L << 30) / (ld * 2)) / 64 * 64;  // rows per piece, half the limit
    if (kc >= 64 && kc < d.K) {
      GemmDesc c = d;
      c.K = (int)kc;
      if (gemm_bf16_dma_ok(layout, c)) {
        const int nbr = gemm_b_rows(false, d);
        for (long k0 = 0; k0 < d.K && k0 < nbr; k0 += kc) {  // rows of B past nbr add zero
          c.K = (int)std::min<long>(kc, d.K - k0);
          c.A = static_cast<const bf16*>(d.A) + k0 * d.lda;
          c.B = static_cast<const bf16*>(d.B) + k0 * d.ldb;
          c.b_rows = (int)std::min<long>(c.K, nbr - k0);
          hipError_t e = gemm_bf16_dma(layout, epi, c, st);
          if (e != hipSuccess) return e;
        }
        return hipSuccess;
      }
    }
  }
  GemmArgs a;
  a.A = d.A; a.B = d.B; a.C = d.C;
  a.M = d.M; a.N = d.N; a.K = d.K;
  a.lda = d.lda; a.ldb = d.ldb; a.ldc = d.ldc;
  a.bias = d.bias; a.R = d.R; a.ldr = d.ldr; a.C2 = d.C2; a.ldc2 = d.ldc2; a.Z = d.Z; a.ldz = d.ldz;
  a.nb = gemm_b_rows(layout == GEMM_NT, d);
  a.res_scale = d.res_scale;
  if (dt == DT_BF16) {
    switch (layout) {
      case GEMM_NT: return dispatch_layout<bf16, GEMM_NT>(epi, a, st);
      case GEMM_NN: return dispatch_layout<bf16, GEMM_NN>(epi, a, st);
      case GEMM_TN: return dispatch_layout<bf16, GEMM_TN>(epi, a, st);
    }
  } else {
    switch (layout) {
      case GEMM_NT: return dispatch_layout<float, GEMM_NT>(epi, a, st);
      case GEMM_NN: return dispatch_layout<float, GEMM_NN>(epi, a, st);
      case GEMM_TN: return dispatch_layout<float, GEMM_TN>(epi, a, st);
    }
  }
  return hipErrorInvalidValue;
}

}  // namespace flglm
