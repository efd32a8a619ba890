// bf16 GEMM for gfx950: C[m, n] (op)= sum_k A(m, k) B(n, k), fp32 accumulate.
//
// Same contract and epilogues as gemm.hip, specialised for the throughput
// path:
//   * 256 x 256 output tile per workgroup, 8 waves (two per SIMD, so one
//     wave's LDS waits are covered by the other's matrix-core work) of
//     128 x 64, reduction stages of 64 double-buffered in LDS (132 KB): a
//     DMA row segment is one full 128-byte line;
//   * operands go from HBM/L2 straight into LDS with buffer loads in LDS-DMA
//     mode (no VGPR staging).  Buffer resources bound each operand, so rows
//     or reduction indices past the end read as zero (ragged token tails);
//   * each operand tile is a set of 1 KB DMA blocks of 8 rows (K-contiguous:
//     rows of 64 reduction indices, read by 16-byte fragment reads;
//     MN-contiguous: k-rows of 64 columns, read by transpose reads
//     (ds_read_b64_tr_b16: lane j of a 16-lane group receives four
//     consecutive-k values of column j when lane s points at
//     (k0 + s/4, c0 + 4 (s % 4)))).  Rows keep their global order inside;
//     which rows share a block, and the blocks' 16- or 32-byte offsets in
//     the bank map, keep the fragment reads free of bank conflicts;
//   * every fragment address is one per-lane base plus a compile-time
//     offset, which keeps the address arithmetic out of the VGPR budget;
//   * an LDS-DMA lane always writes to base + 16 * lane, so the placement is
//     chosen through the source addresses;
//   * one barrier per stage, placed between the two 32-wide halves: the
//     second half's fragments are already in registers when the barrier
//     releases the slot, so the next stage's loads and fragment reads overlap
//     matrix-core work.
#include <algorithm>

#include "common.h"
#include "kernels.h"

namespace flglm {
namespace {

constexpr int kBM = 256, kBN = 256, kBK = 64, kStages = 2, kThr = 512, kWaves = 8;
// waves: 2 along M x 4 along N, each 128 x 64 (8 x 4 tiles of 16 x 16)
constexpr int kWTM = 8, kWTN = 4;
// LDS region of one operand tile: the MN-contiguous layout pads each 1 KB
// DMA block to 1056 bytes (33 KB in all)
constexpr int kRegionElems = 16896, kMBlock = 528, kMCol = 8 * kMBlock, kKBlock = 520;
typedef short i16x4 __attribute__((ext_vector_type(4)));
#define LDS_AS __attribute__((address_space(3)))

struct G2Args {
  const bf16* A;
  const bf16* B;
  void* C;
  int M, N, K;
  long lda, ldb, ldc;
  const bf16* bias;
  const bf16* R;
  long ldr;
  bf16* C2;
  long ldc2;
  const bf16* Z;
  long ldz;
  // Split reduction for the last, partial round of tiles: the final `tail`
  // tiles are cut into `splits` reduction slices whose fp32 partial
  // accumulators go to `part`; a second launch (fixup = 1) sums them in a
  // fixed order and runs the epilogue.
  float* part;
  int tail, splits, fixup;
  int nb;  // rows of B that exist (see GemmDesc::b_rows)
  float res_scale;
  // EPI_GELU_BWD: per 256-row tile, the column sums of the stored C (fp32
  // [tiles_m][N]), or null
  float* colsum;
};


__device__ __forceinline__ void dma16(i32x4 rs, uint32_t lds_inst_base, uint32_t voff) {
  dma_lds<16>(rs, lds_inst_base, voff);
}

// Per-lane source byte offsets (reduction index 0) of DMA instruction inst
// (0..31) of an operand tile.
// K-contiguous tile [256 rows][64]: 32 DMA blocks of 8 rows of 128 bytes at a
// stride of 1040 bytes, every row read in address order (as below).  Row
// r = 16 q + t sits in block b = (t & 7) + 8 (q >> 2), row 2 (q & 3) + (t >> 3):
// the 16 rows that one 16-lane fragment read touches (one 16-row group q)
// sit in 8 blocks (16-byte shifts 16 b) at two row parities, i.e. on 16
// distinct bank groups for 16 consecutive lanes.  The LDS serves a 16-byte
// read per cycle to the 16 lanes sharing lane bit 5 and the parity of bits
// 2-4, for which these reads are 2-way conflicted; a placement free of that
// (1056-byte blocks, row parities 512 bytes apart) measured no faster.
// Instruction inst fills block inst.
__device__ __forceinline__ uint32_t k_src(long ld, int inst, int lane) {
  const int slot = lane >> 3;
  const int row = 16 * (4 * (inst >> 3) + (slot >> 1)) + (inst & 7) + 8 * (slot & 1);
  return (uint32_t)(row * ld + (lane & 7) * 8) * 2u;
}
// MN-contiguous tile: 4 column blocks of 64 columns (kMCol elements each),
// each 8 DMA blocks b of 8 k-rows of 128 bytes, at a stride of 1056 bytes.
// Every k-row is one DMA row segment read in address order: the texture
// addresser handles a permuted segment several times slower (counted as
// SQ_VMEM_TA_ADDR_FIFO_FULL), so bank spreading comes from where whole rows
// go instead of a swizzle inside them.  k-row k (k = c + 4 s0 + 8 p + 16 s1 +
// 32 h, each digit a bit) sits in block b = c + 4 h, row r = p + 2 s0 + 4 s1.
// A transpose read serves 32 lanes per cycle: k-rows kb .. kb+3 and
// kb+8 .. kb+11 (kb = 0, 4, 16, 20, + 32), 32 bytes each; these sit in four
// blocks (32-byte shifts 32 b) at two row parities: eight distinct bank
// groups.  Instruction inst fills block inst % 8 of column block inst / 8.
__device__ __forceinline__ uint32_t m_src(long ld, int inst, int lane) {
  const int blk = inst >> 3, b = inst & 7;
  const int krow = (b & 3) + 4 * ((lane >> 4) & 1) + 8 * ((lane >> 3) & 1) + 16 * (lane >> 5) + 32 * (b >> 2);
  return (uint32_t)((long)krow * ld + blk * 64 + (lane & 7) * 8) * 2u;
}
// LDS byte offset, inside an operand region, of DMA instruction inst
__device__ __forceinline__ uint32_t k_dst(int inst) { return (uint32_t)inst * (2u * kKBlock); }
__device__ __forceinline__ uint32_t m_dst(int inst) { return (uint32_t)((inst >> 3) * kMCol + (inst & 7) * kMBlock) * 2u; }

// Per-lane fragment bases (element offsets inside one operand tile).
// K-contiguous: fragment j of a wave (rows row0 + 16 j, row0 a multiple of
// 64), reduction half c: lane (fr, fg) reads chunk fg + 4 c of row
// row0 + 16 j + fr.
__device__ __forceinline__ int frag_k_base(int row0, int fr, int fg) {
  return (fr & 7) * kKBlock + 64 * (fr >> 3) + 8 * fg + 8 * kKBlock * (row0 >> 6);
}
// MN-contiguous: fragment j (columns col0 + 16 j), reduction half c: lane s
// of a 16-lane group points at k-row 8 g + s / 4 (block s / 4, row
// (g & 1) + 4 (g >> 1)), columns 4 (s % 4) of group j % 4 of column block
// col0 / 64 + j / 4; the second read is k + 4 (row + 2), half c = k + 32
// (block + 4).
__device__ __forceinline__ int frag_m_base(int col0, int fr, int fg) {
  return (col0 >> 6) * kMCol + (fr >> 2) * kMBlock + ((fg & 1) + 4 * (fg >> 1)) * 64 + 4 * (fr & 3);
}
__device__ __forceinline__ bf16x8 frag_k(const bf16* tile, int base, int c, int j) {
  return __builtin_bit_cast(bf16x8, ld16(tile + base + 8 * kKBlock * (j >> 2) + 128 * (j & 3) + 32 * c));
}
__device__ __forceinline__ bf16x8 frag_m(const bf16* tile, int base, int c, int j) {
  const bf16* p = tile + base + 16 * (j & 3) + kMCol * (j >> 2) + 4 * kMBlock * c;
  i16x4 a = __builtin_amdgcn_ds_read_tr16_b64_v4i16((LDS_AS i16x4*)(p));
  i16x4 b = __builtin_amdgcn_ds_read_tr16_b64_v4i16((LDS_AS i16x4*)(p + 128));
  return __builtin_bit_cast(bf16x8, __builtin_shufflevector(a, b, 0, 1, 2, 3, 4, 5, 6, 7));
}

// tanh-form GeLU via the logistic function: 0.5 (1 + tanh u) = sigma(2u), so
//   gelu(z)  = z sigma(2u),  u = sqrt(2/pi) (z + 0.044715 z^3)
//   gelu'(z) = sigma(2u) + 2 z sigma(2u) (1 - sigma(2u)) sqrt(2/pi) (1 + 3 * 0.044715 z^2)
// with sigma(v) = 1 / (1 + 2^(-v log2 e)) from the hardware exp2 and reciprocal
// (about 1 ulp each; exp2 saturates to 0 / inf, which gives sigma = 1 / 0).
__device__ __forceinline__ float sigmoid2u(float z) {
  const float c2 = 2.0f * 0.7978845608028654f * kLog2e, a = 0.044715f;
  const float e = __builtin_amdgcn_exp2f(-c2 * (z + a * z * z * z));
  return __builtin_amdgcn_rcpf(1.0f + e);
}
__device__ __forceinline__ float gelu2(float z) { return z * sigmoid2u(z); }
__device__ __forceinline__ float gelu2_grad(float z) {
  const float c = 0.7978845608028654f, a = 0.044715f;
  const float s = sigmoid2u(z);
  return s + 2.0f * c * z * s * (1.0f - s) * (1.0f + 3.0f * a * z * z);
}

// Tile order: workgroup wg runs on XCD wg % 8, and each XCD takes a contiguous
// range of tile ids, walked column by column inside bands of kGroupM tile rows.
// With 4-row bands the 32 tiles one XCD holds at a time span 4 row panels of A
// and 8 column panels of B; for the token-major products (forward, dgrad)
// that is 1.5-3 % faster than 8-row bands (16 rows: 5-18 % slower than 8).
// The weight gradient (both operands MN-contiguous) measures 0.6 % faster
// with 8.
template <int kGroupM>
__device__ __forceinline__ void tile_coords2(int wg, int nwg, int tiles_m, int tiles_n, int& tm, int& tn) {
  constexpr int kXcd = 8;
  const int q = nwg / kXcd, r = nwg % kXcd;
  const int x = wg % kXcd, j = wg / kXcd;
  const int id = (x < r) ? x * (q + 1) + j : r * (q + 1) + (x - r) * q + j;
  const int per_group = kGroupM * tiles_n;
  const int group = id / per_group;
  const int first_m = group * kGroupM;
  const int gsize = min(tiles_m - first_m, kGroupM);
  const int in_group = id % per_group;
  tm = first_m + in_group % gsize;
  tn = in_group / gsize;
}

// Bare workgroup barrier: a fence would also wait for DMA stages in flight.
__device__ __forceinline__ void wg_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Epilogue of one 256 x 256 tile from the wave accumulators acc[i][j]
// (wave tile rows 128 (wave & 1) + 16 j, columns 64 (wave >> 1) + 16 i), with
// the LDS at stg (at least 128 KB, free: every wave is past its operand
// reads) as staging.  The accumulators of one 128-row half of the tile go to
// LDS as fp32 ([128][256]); then a lane owns eight consecutive columns
// (group cg = lane % 32) and the two halves of a wave take alternate rows,
// so bias, residual, GeLU-input and output rows are read and written
// contiguously, 16 bytes per lane, two rows per wave instruction (a lane of
// the matrix core holds 4 columns of 16 different rows, which as direct
// stores cost more than the reduction for K = 4096; a CU's store
// instructions cost about the same at 8 and at 16 bytes per lane, so the
// wide form halves the row loop's memory instructions).  Staging puts
// 16-byte chunk c of row r at c ^ (r & 15) ^ ((c >> 4) & 1): the row writes
// of the matrix-core lanes and the 16-lane reads of even (or odd) chunks
// both hit 16 distinct bank groups.
__device__ __forceinline__ int stg_swz(int r, int c) { return c ^ (r & 15) ^ ((c >> 4) & 1); }

template <int EPI, int BATCH>
__device__ __forceinline__ void tile_epilogue(const G2Args& p, const f32x4 (&acc)[kWTN][kWTM], float* stg, int tm,
                                              int m0, int n0, int tid) {
  asm volatile("" : "+v"(tid));  // keeps the epilogue's per-lane values out of the main loop's live range
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = wave & 1, wn = wave >> 1;
  const int fr = lane & 15, fg = lane >> 4;
  const int sh = lane >> 5, cg = lane & 31;
  const int n = n0 + 8 * cg;
  float bias[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  // EPI_GELU_BWD with colsum: this lane's eight columns over its rows (the
  // stored, rounded values), in row order
  float csum[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  if constexpr (EPI == EPI_BIAS || EPI == EPI_BIAS_RES || EPI == EPI_BIAS_GELU) {
    Vec8<bf16> b;
    b.load(p.bias + n);
#pragma unroll
    for (int e = 0; e < 8; ++e) bias[e] = b.get(e);
  }
#pragma unroll
  for (int half = 0; half < 2; ++half) {
    const int mbase = m0 + half * 128 + wave;
    if (wm == half) {
#pragma unroll
      for (int j = 0; j < kWTM; ++j) {
        const int r = 16 * j + fr;
#pragma unroll
        for (int i = 0; i < kWTN; ++i) {
          const int c = (wn * 64 + 16 * i + 4 * fg) >> 2;
          st16(stg + r * 256 + (stg_swz(r, c) << 2), __builtin_bit_cast(u32x4, acc[i][j]));
        }
      }
    }
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    wg_barrier();
    // Rows wave + 8 q, q = 2 t + sh (t = 0..7), in batches of row pairs
    // whose global loads are issued together before their first use.
    constexpr int kB = BATCH / 2 > 0 ? BATCH / 2 : 1;
#pragma unroll
    for (int t0 = 0; t0 < 8; t0 += kB) {
      Vec8<bf16> ext[kB];
      Vec8<float> cacc[kB];
#pragma unroll
      for (int u = 0; u < kB; ++u) {
        const long m = mbase + (2 * (t0 + u) + sh) * kWaves;
        if (m < p.M) {
          if constexpr (EPI == EPI_BIAS_RES || EPI == EPI_RES) ext[u].load(p.R + m * p.ldr + n);
          if constexpr (EPI == EPI_GELU_BWD) ext[u].load(p.Z + m * p.ldz + n);
          if constexpr (EPI == EPI_ACC_F32) cacc[u].load(static_cast<float*>(p.C) + m * p.ldc + n);
        }
      }
#pragma unroll
      for (int u = 0; u < kB; ++u) {
        const int q = 2 * (t0 + u) + sh;
        const int r = wave + q * kWaves;
        const long m = mbase + q * kWaves;
        if (m >= p.M) break;
        const u32x4 raw0 = ld16(stg + r * 256 + (stg_swz(r, 2 * cg) << 2));
        const u32x4 raw1 = ld16(stg + r * 256 + (stg_swz(r, 2 * cg + 1) << 2));
        float v[8];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          v[e] = __uint_as_float(raw0[e]) + bias[e];
          v[4 + e] = __uint_as_float(raw1[e]) + bias[4 + e];
        }
        if constexpr (EPI == EPI_ACC_F32) {
          float o[8];
#pragma unroll
          for (int e = 0; e < 8; ++e) o[e] = cacc[u].get(e) + v[e];
          cacc[u].set(o);
          cacc[u].store(static_cast<float*>(p.C) + m * p.ldc + n);
        } else {
          if constexpr (EPI == EPI_BIAS_RES || EPI == EPI_RES) {
#pragma unroll
            for (int e = 0; e < 8; ++e) v[e] += p.res_scale * ext[u].get(e);
          }
          if constexpr (EPI == EPI_GELU_BWD) {
#pragma unroll
            for (int e = 0; e < 8; ++e) v[e] *= gelu2_grad(ext[u].get(e));
          }
          Vec8<bf16> o;
          o.set(v);
          if (EPI != EPI_BIAS_GELU || p.C) o.store(static_cast<bf16*>(p.C) + m * p.ldc + n);
          if constexpr (EPI == EPI_GELU_BWD) {
#pragma unroll
            for (int e = 0; e < 8; ++e) csum[e] += o.get(e);
          }
          if constexpr (EPI == EPI_BIAS_GELU) {
            float g[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) g[e] = gelu2(v[e]);
            Vec8<bf16> og;
            og.set(g);
            og.store(p.C2 + m * p.ldc2 + n);
          }
        }
      }
    }
    // the second half, or the next tile's loads, overwrite the staging area
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    wg_barrier();
  }
  if constexpr (EPI == EPI_GELU_BWD) {
    if (p.colsum) {
      // the sixteen half-waves' partial column sums, added in (wave, half)
      // order (the operand tiles are free: every wave passed the barrier)
      float* cs = stg;
      float* mine = cs + (wave * 2 + sh) * kBN + 8 * cg;
      st16(mine, __builtin_bit_cast(u32x4, f32x4{csum[0], csum[1], csum[2], csum[3]}));
      st16(mine + 4, __builtin_bit_cast(u32x4, f32x4{csum[4], csum[5], csum[6], csum[7]}));
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
      wg_barrier();
      if (tid < kBN) {
        float t = 0.f;
#pragma unroll
        for (int w2 = 0; w2 < 2 * kWaves; ++w2) t += cs[w2 * kBN + tid];
        p.colsum[(long)tm * p.N + n0 + tid] = t;
      }
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
      wg_barrier();  // the next tile's loads overwrite cs
    }
  }
}

// Rows of the epilogue whose global reads are issued together: 16 for the
// residual epilogues (a half's whole share: 6 % faster on the 41447 x 4096 x
// 4096 output projection than 8), 8 elsewhere (16 measured no faster), 4 for
// the fp32 accumulator.
template <int EPI>
constexpr int epi_batch() { return (EPI == EPI_BIAS_RES || EPI == EPI_RES) ? 16 : EPI == EPI_ACC_F32 ? 4 : 8; }

template <bool AK, bool BKc, int EPI, int BATCH = epi_batch<EPI>()>
__global__ void __launch_bounds__(kThr) gemm_bf16_kernel(G2Args p) {
  __shared__ __attribute__((aligned(1024))) bf16 smem[kStages][2][kRegionElems];  // [stage][A/B]

  const int tiles_m = (p.M + kBM - 1) / kBM, tiles_n = p.N / kBN;
  const int ntiles = tiles_m * tiles_n;
  const int nk = (p.K + kBK - 1) / kBK;
  const int full = ntiles - p.tail;
  const int nwork = p.fixup ? p.tail : full + p.tail * p.splits;
  // Persistent: one workgroup per CU walks the work items (whole tiles, then
  // the reduction slices of the tail tiles); a tile's epilogue stores drain
  // while the next item's first stages load.
  for (int wi = blockIdx.x; wi < nwork; wi += gridDim.x) {
  int t, kt0 = 0, kt1 = nk, slice = -1;
  if (p.fixup) {
    t = full + wi;
  } else if (wi < full) {
    t = wi;
  } else {
    slice = wi - full;
    t = full + slice / p.splits;
    const int per = (nk + p.splits - 1) / p.splits;
    kt0 = min(nk, (slice % p.splits) * per);
    kt1 = min(nk, kt0 + per);
  }
  // Per-lane values are rederived in every tile (the opaque copy keeps the
  // compiler from hoisting them out of the tile loop, where they would stay
  // live across the whole body and spill).
  int tid = threadIdx.x;
  asm volatile("" : "+v"(tid));
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = wave & 1, wn = wave >> 1;  // wave tile: rows wm*128.., columns wn*64..
  const int fr = lane & 15, fg = lane >> 4;
  int tm, tn;
  tile_coords2<(AK || BKc) ? 4 : 8>(t, ntiles, tiles_m, tiles_n, tm, tn);
  const int m0 = tm * kBM, n0 = tn * kBN;

  // Resources: K-contiguous -> base at the tile's first row, bound = its
  // valid rows; MN-contiguous -> base at the tile's first column, bound = the
  // rest of the buffer (reduction indices >= K read as zero).
  i32x4 ra, rb;
  if constexpr (AK) {
    const int rows = min(kBM, p.M - m0);
    ra = buf_rsrc(p.A + (long)m0 * p.lda, (uint32_t)((long)rows * p.lda * 2));
  } else {
    ra = buf_rsrc(p.A + m0, (uint32_t)(((long)p.K * p.lda - m0) * 2));
  }
  if constexpr (BKc) {
    // rows of B past p.nb (a padded N) do not exist: num_records 0 for a
    // tile wholly past them, so nothing is read there
    const int rows = p.nb > n0 ? min(kBN, p.nb - n0) : 0;
    rb = buf_rsrc(p.B + (long)n0 * p.ldb, (uint32_t)((long)rows * p.ldb * 2));
  } else {
    rb = buf_rsrc(p.B + n0, (uint32_t)(((long)p.nb * p.ldb - n0) * 2));
  }
  // DMA bookkeeping.  Each stage takes 32 DMA instructions per operand.
  // Forward and dgrad: every wave issues 4 per operand, instruction i of
  // wave w being instruction 8 i + w of the tile.  Weight gradient: waves 0-3
  // issue 8 per operand (instruction 4 i + w) and waves 4-7 none.  Waves w
  // and w + 4 share a SIMD, so each SIMD then pairs a loading wave with one
  // that only computes: a load stalled on the texture unit's address queue
  // holds up only the loading wave's matrix instructions while the other
  // wave's instructions keep the matrix core busy (3 % faster on the wgrad; the forward
  // and dgrad products measured within +-1 %).  k_dst / m_dst are linear in
  // the instruction index for these wave numbers, so a wave adds its own
  // offset once.  The per-lane source offsets are fixed up to the stage's
  // reduction offset, added per stage.
  constexpr bool kLoaders = !AK && !BKc;
  constexpr int kDmaPer = kLoaders ? 8 : 4;          // per operand per stage per loading wave
  constexpr int kDmaStride = 32 / kDmaPer;           // tile instruction stride between a wave's DMAs
  const bool loader = !kLoaders || wave < 4;
  const int wq = kLoaders ? (wave & 3) : wave;
  const uint32_t lds0 = FL_LDS_ADDR(&smem[0][0][0]);
  const uint32_t lds_a = __builtin_amdgcn_readfirstlane(lds0 + (AK ? k_dst(wq) : m_dst(wq)));
  const uint32_t lds_b =
      __builtin_amdgcn_readfirstlane(lds0 + kRegionElems * 2 + (BKc ? k_dst(wq) : m_dst(wq)));
  uint32_t voa[kDmaPer], vob[kDmaPer];
#pragma unroll
  for (int i = 0; i < kDmaPer; ++i) {
    voa[i] = AK ? k_src(p.lda, i * kDmaStride + wq, lane) : m_src(p.lda, i * kDmaStride + wq, lane);
    vob[i] = BKc ? k_src(p.ldb, i * kDmaStride + wq, lane) : m_src(p.ldb, i * kDmaStride + wq, lane);
  }
  // byte offset of reduction index k0 along each operand
  auto kstep_a = [&](int k0) { return AK ? (uint32_t)k0 * 2u : (uint32_t)((long)k0 * p.lda * 2); };
  auto kstep_b = [&](int k0) { return BKc ? (uint32_t)k0 * 2u : (uint32_t)((long)k0 * p.ldb * 2); };
  // DMA instruction g (A 0 .. kDmaPer-1, then B) of this wave for stage kt
  auto dma_one = [&](int kt, int g) {
    const uint32_t slot_off = (uint32_t)(kt & (kStages - 1)) * (2 * kRegionElems * 2);
    if (g < kDmaPer) {
      const int o = kDmaStride * g;
      dma16(ra, lds_a + slot_off + (AK ? k_dst(o) : m_dst(o)), voa[g] + kstep_a(kt * kBK));
    } else {
      const int o = kDmaStride * (g - kDmaPer);
      dma16(rb, lds_b + slot_off + (BKc ? k_dst(o) : m_dst(o)), vob[g - kDmaPer] + kstep_b(kt * kBK));
    }
  };
  auto issue = [&](int kt) {
    if (loader) {
#pragma unroll
      for (int g = 0; g < 2 * kDmaPer; ++g) dma_one(kt, g);
    }
  };
  const int abase = AK ? frag_k_base(wm * 128, fr, fg) : frag_m_base(wm * 128, fr, fg);
  const int bbase = BKc ? frag_k_base(wn * 64, fr, fg) : frag_m_base(wn * 64, fr, fg);

  f32x4 acc[kWTN][kWTM];
#pragma unroll
  for (int i = 0; i < kWTN; ++i)
#pragma unroll
    for (int j = 0; j < kWTM; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  auto rd_a = [&](int slot, int c, int j) {
    const bf16* as = smem[slot][0];
    return AK ? frag_k(as, abase, c, j) : frag_m(as, abase, c, j);
  };
  auto rd_b = [&](int slot, int c, int i) {
    const bf16* bs = smem[slot][1];
    return BKc ? frag_k(bs, bbase, c, i) : frag_m(bs, bbase, c, i);
  };
  // fragments of reduction half c of the stage in slot `slot`
  auto load_frags = [&](int slot, int c, bf16x8 (&af)[kWTM], bf16x8 (&bf)[kWTN]) {
#pragma unroll
    for (int i = 0; i < kWTN; ++i) bf[i] = rd_b(slot, c, i);
#pragma unroll
    for (int j = 0; j < kWTM; ++j) af[j] = rd_a(slot, c, j);
  };
  auto mma_all = [&](const bf16x8 (&af)[kWTM], const bf16x8 (&bf)[kWTN]) {
#pragma unroll
    for (int j = 0; j < kWTM; ++j)
#pragma unroll
      for (int i = 0; i < kWTN; ++i) acc[i][j] = mma16(bf[i], af[j], acc[i][j]);
  };
  // bare barrier: a fence would also wait for the younger stage in flight
  auto barrier = [&]() {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
  };

  if (p.fixup) {
    // sum the tile's reduction slices in slice order (deterministic)
    const float* src = p.part + (long)(t - full) * p.splits * (kWTN * kWTM * kThr * 4);
    for (int c = 0; c < p.splits; ++c) {
#pragma unroll
      for (int i = 0; i < kWTN; ++i)
#pragma unroll
        for (int j = 0; j < kWTM; ++j)
          acc[i][j] += __builtin_bit_cast(f32x4, ld16(src + ((long)(c * kWTN * kWTM + i * kWTM + j) * kThr + tid) * 4));
    }
  } else if (kt1 > kt0) {
  // Stage kt lives in slot kt % 2.  Prologue: stages 0 and 1 in flight; once
  // stage 0 is visible, read its first half.
  issue(kt0);
  if (kt1 - kt0 > 1) {
    issue(kt0 + 1);
    // the older stage's loads done: at most one stage (2 kDmaPer) in flight
    if constexpr (kLoaders)
      asm volatile("s_waitcnt vmcnt(16)" ::: "memory");
    else
      asm volatile("s_waitcnt vmcnt(8)" ::: "memory");
  } else {
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  }
  barrier();
  bf16x8 fa0[kWTM], fb0[kWTN], fa1[kWTM], fb1[kWTN];
  load_frags(kt0 & 1, 0, fa0, fb0);
  // Main loop, one stage per iteration, in two halves of 32 reductions.  The
  // issue order is fixed by scheduling barriers: each group of four matrix
  // instructions (one A fragment against the four B fragments) is preceded
  // by one or two fragment reads for the next half and, in the second half,
  // by one (each wave) or two (loading waves of the wgrad) of the DMA
  // instructions for stage kt + 2, so the memory pipes are fed steadily
  // instead of in bursts that stall issue.
  // The last stage is peeled so that every path through the body passes the
  // barrier (the compiler then never waits for next-half reads early).
  for (int kt = kt0; kt < kt1 - 1; ++kt) {
    const int slot = kt & 1;
#pragma unroll
    for (int j = 0; j < kWTM; ++j) {
      fa1[j] = rd_a(slot, 1, j);
      if (j < kWTN) fb1[j] = rd_b(slot, 1, j);
      __builtin_amdgcn_sched_barrier(0);
      __builtin_amdgcn_s_setprio(1);  // the matrix group wins issue over the other wave's memory ops
#pragma unroll
      for (int i = 0; i < kWTN; ++i) acc[i][j] = mma16(fb0[i], fa0[j], acc[i][j]);
      __builtin_amdgcn_s_setprio(0);
      __builtin_amdgcn_sched_barrier(0);
    }
    // stage kt+1 landed (own loads) and every wave has finished reading
    // slot kt: refill it with stage kt+2, read stage kt+1's first half
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    barrier();
    const bool more = kt + 2 < kt1;
#pragma unroll
    for (int j = 0; j < kWTM; ++j) {
      if (more && loader) {
        dma_one(kt + 2, (kDmaPer / 4) * j);
        if constexpr (kLoaders) dma_one(kt + 2, 2 * j + 1);
      }
      fa0[j] = rd_a(slot ^ 1, 0, j);
      if (j < kWTN) fb0[j] = rd_b(slot ^ 1, 0, j);
      __builtin_amdgcn_sched_barrier(0);
      __builtin_amdgcn_s_setprio(1);
#pragma unroll
      for (int i = 0; i < kWTN; ++i) acc[i][j] = mma16(fb1[i], fa1[j], acc[i][j]);
      __builtin_amdgcn_s_setprio(0);
      __builtin_amdgcn_sched_barrier(0);
    }
  }
  load_frags((kt1 - 1) & 1, 1, fa1, fb1);
  mma_all(fa0, fb0);
  mma_all(fa1, fb1);
  }
  if (slice >= 0) {
    // a reduction slice of a tail tile: store the partial accumulators
    // ([slice][i][j][thread][4], coalesced) and move on
    float* dst = p.part + (long)slice * (kWTN * kWTM * kThr * 4);
#pragma unroll
    for (int i = 0; i < kWTN; ++i)
#pragma unroll
      for (int j = 0; j < kWTM; ++j)
        st16(dst + ((long)(i * kWTM + j) * kThr + tid) * 4, __builtin_bit_cast(u32x4, acc[i][j]));
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    barrier();  // every wave is done with the operand tiles before the next item's loads
    continue;
  }

  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  barrier();  // every wave is done with the operand tiles
  tile_epilogue<EPI, BATCH>(p, acc, reinterpret_cast<float*>(&smem[0][0][0]), tm, m0, n0, tid);
  }
}

// fp32 partial accumulators of one 256 x 256 tile slice
constexpr size_t kSliceBytes = (size_t)kBM * kBN * 4;

// Compute units of the current device (one persistent workgroup each; a
// multiple of the 8 XCDs on MI355X, which the tile order relies on).
int num_cus() {
  static int cached[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) dev = 0;
  if (cached[dev] == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
    cached[dev] = n - n % 8 > 0 ? n - n % 8 : n;
  }
  return cached[dev];
}

template <bool AK, bool BKc, int EPI>
hipError_t launch2(const GemmDesc& d, hipStream_t st) {
  G2Args a;
  a.A = (const bf16*)d.A; a.B = (const bf16*)d.B; a.C = d.C;
  a.M = d.M; a.N = d.N; a.K = d.K; a.lda = d.lda; a.ldb = d.ldb; a.ldc = d.ldc;
  a.bias = (const bf16*)d.bias; a.R = (const bf16*)d.R; a.ldr = d.ldr;
  a.C2 = (bf16*)d.C2; a.ldc2 = d.ldc2; a.Z = (const bf16*)d.Z; a.ldz = d.ldz;
  a.part = d.part; a.tail = 0; a.splits = 1; a.fixup = 0;
  a.nb = gemm_b_rows(BKc, d);
  a.res_scale = d.res_scale;
  a.colsum = EPI == EPI_GELU_BWD ? d.colsum : nullptr;
  const int tiles = ((d.M + kBM - 1) / kBM) * (d.N / kBN);
  if (tiles == 0) return hipSuccess;
  const int cus = num_cus();
  // A last round that would leave three quarters of the CUs idle is cut
  // into reduction slices (at least 4 stages each) spread over all CUs.
  // Measured on MI355X: worth it from 128 stages (K = 8192) on; below that
  // the partial stores and the fixup launch cost more than the idle CUs.
  const int rem = tiles % cus, nk = (d.K + kBK - 1) / kBK;
  if (d.part && rem > 0 && 4 * rem <= cus && nk >= 128) {
    int splits = std::min(std::min(cus / rem, nk / 4), 16);
    while (splits > 1 && (size_t)rem * splits * kSliceBytes > d.part_bytes) --splits;
    if (splits > 1) {
      a.tail = rem;
      a.splits = splits;
    }
  }
  const int items = tiles - a.tail + a.tail * a.splits;
  hipLaunchKernelGGL((gemm_bf16_kernel<AK, BKc, EPI>), dim3(items < cus ? items : cus), dim3(kThr), 0, st, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || a.tail == 0) return e;
  a.fixup = 1;
  hipLaunchKernelGGL((gemm_bf16_kernel<AK, BKc, EPI>), dim3(a.tail), dim3(kThr), 0, st, a);
  return hipGetLastError();
}

}  // namespace

// One slice per compute unit of an MI355X (256); launches split only as far
// as the scratch they are given allows.
size_t gemm_part_bytes() { return (size_t)256 * kSliceBytes; }

// Shapes the DMA kernel takes: N a multiple of 256, K-contiguous operands
// with K a multiple of 64, and every buffer offset below 2^31 bytes.
bool gemm_bf16_dma_ok(GemmLayout layout, const GemmDesc& d) {
  if (d.N % kBN != 0 || d.M <= 0) return false;
  const bool ak = layout != GEMM_TN, bk = layout == GEMM_NT;
  if ((ak || bk) && d.K % kBK != 0) return false;
  const long lim = 1L << 31;
  if (!ak && (long)d.K * d.lda * 2 >= lim) return false;
  if (!bk && (long)d.K * d.ldb * 2 >= lim) return false;
  if (ak && (long)kBM * d.lda * 2 >= lim) return false;
  if (bk && (long)kBN * d.ldb * 2 >= lim) return false;
  return true;
}

bool gemm_fuses_colsum(DType dt, GemmLayout layout, int epi, const GemmDesc& d) {
  return dt == DT_BF16 && layout == GEMM_NN && epi == EPI_GELU_BWD && kBM == kColsumRows &&
         gemm_bf16_dma_ok(layout, d);
}

hipError_t gemm_bf16_dma(GemmLayout layout, int epi, const GemmDesc& d, hipStream_t st) {
  switch (layout) {
    case GEMM_NT:
      switch (epi) {
        case EPI_STORE: return launch2<true, true, EPI_STORE>(d, st);
        case EPI_BIAS: return launch2<true, true, EPI_BIAS>(d, st);
        case EPI_BIAS_RES: return launch2<true, true, EPI_BIAS_RES>(d, st);
        case EPI_BIAS_GELU: return launch2<true, true, EPI_BIAS_GELU>(d, st);
      }
      break;
    case GEMM_NN:
      switch (epi) {
        case EPI_STORE: return launch2<true, false, EPI_STORE>(d, st);
        case EPI_GELU_BWD: return launch2<true, false, EPI_GELU_BWD>(d, st);
        case EPI_RES: return launch2<true, false, EPI_RES>(d, st);
      }
      break;
    case GEMM_TN:
      if (epi == EPI_ACC_F32) return launch2<false, false, EPI_ACC_F32>(d, st);
      break;
  }
  return hipErrorInvalidValue;
}

}  // namespace flglm
