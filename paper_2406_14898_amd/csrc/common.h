// Device-side building blocks shared by every kernel of the library:
// element types, 16-byte vector memory ops, bf16 conversion, and the one
// matrix-core primitive every contraction is written against.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace flglm {

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x8 __attribute__((ext_vector_type(8)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr float kLog2e = 1.4426950408889634f;

// ---------------------------------------------------------------------------
// Scalar conversions.  float -> bf16 rounds to nearest even (the hardware
// conversion on gfx950); bf16 -> float is exact.
// ---------------------------------------------------------------------------
__device__ __forceinline__ float to_f32(float v) { return v; }
__device__ __forceinline__ float to_f32(bf16 v) { return static_cast<float>(v); }
template <typename T> __device__ __forceinline__ T from_f32(float v);
template <> __device__ __forceinline__ float from_f32<float>(float v) { return v; }
template <> __device__ __forceinline__ bf16 from_f32<bf16>(float v) { return static_cast<bf16>(v); }

// ---------------------------------------------------------------------------
// Eight-element fragments: bf16x8 is one 16-byte register quad, the fp32
// variant is two.  Fragments are the unit of LDS traffic for the matrix core.
// ---------------------------------------------------------------------------
template <typename T> struct Frag;
template <> struct Frag<bf16> { typedef bf16x8 type; };
template <> struct Frag<float> { typedef f32x8 type; };
template <typename T> using frag_t = typename Frag<T>::type;

// One 16x16 output tile, reduction over 32 "slots".  Lane l supplies row
// (l % 16) of the first operand and column (l % 16) of the second operand,
// each as eight reduction slots; the result lane l holds column (l % 16),
// rows 4*(l/16) .. 4*(l/16)+3.  Any assignment of slots to reduction indices
// is valid as long as both operands use the same one, which lets callers
// permute the reduction order freely (e.g. to consume accumulator layouts
// directly).  bf16 uses one 16x16x32 MFMA; fp32 uses eight 16x16x4 MFMAs,
// slot j of every lane going to the j-th instruction.
__device__ __forceinline__ f32x4 mma16(const bf16x8& a, const bf16x8& b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ f32x4 mma16(const f32x8& a, const f32x8& b, f32x4 c) {
#pragma unroll
  for (int j = 0; j < 8; ++j) c = __builtin_amdgcn_mfma_f32_16x16x4f32(a[j], b[j], c, 0, 0, 0);
  return c;
}

// ---------------------------------------------------------------------------
// Vector memory helpers (16-byte granules).
// ---------------------------------------------------------------------------
__device__ __forceinline__ u32x4 ld16(const void* p) { return *reinterpret_cast<const u32x4*>(p); }
__device__ __forceinline__ void st16(void* p, const u32x4& v) { *reinterpret_cast<u32x4*>(p) = v; }
__device__ __forceinline__ u32x2 ld8(const void* p) { return *reinterpret_cast<const u32x2*>(p); }
__device__ __forceinline__ void st8(void* p, const u32x2& v) { *reinterpret_cast<u32x2*>(p) = v; }

// Eight consecutive elements of type T at p (16 bytes for bf16, 32 for fp32).
template <typename T> struct Vec8;
template <> struct Vec8<bf16> {
  u32x4 r;
  __device__ __forceinline__ void load(const bf16* p) { r = ld16(p); }
  __device__ __forceinline__ void store(bf16* p) const { st16(p, r); }
  __device__ __forceinline__ void zero() { r = u32x4{0, 0, 0, 0}; }
  // Opaque redefinition: values converted from the vector before this point
  // are not reused after it (the compiler re-reads the packed registers).
  __device__ __forceinline__ void settle() { asm volatile("" : "+v"(r)); }
  __device__ __forceinline__ float get(int i) const {
    uint32_t w = r[i >> 1];
    return __uint_as_float((i & 1) ? (w & 0xffff0000u) : (w << 16));
  }
  __device__ __forceinline__ bf16x8 frag() const { return __builtin_bit_cast(bf16x8, r); }
  __device__ __forceinline__ void set(const float (&v)[8]) {
    bf16x8 b = {from_f32<bf16>(v[0]), from_f32<bf16>(v[1]), from_f32<bf16>(v[2]), from_f32<bf16>(v[3]),
                from_f32<bf16>(v[4]), from_f32<bf16>(v[5]), from_f32<bf16>(v[6]), from_f32<bf16>(v[7])};
    r = __builtin_bit_cast(u32x4, b);
  }
};
template <> struct Vec8<float> {
  u32x4 r0, r1;
  __device__ __forceinline__ void load(const float* p) { r0 = ld16(p); r1 = ld16(p + 4); }
  __device__ __forceinline__ void store(float* p) const { st16(p, r0); st16(p + 4, r1); }
  __device__ __forceinline__ void zero() { r0 = u32x4{0, 0, 0, 0}; r1 = r0; }
  __device__ __forceinline__ void settle() { asm volatile("" : "+v"(r0), "+v"(r1)); }
  __device__ __forceinline__ float get(int i) const { return __uint_as_float(i < 4 ? r0[i & 3] : r1[i & 3]); }
  __device__ __forceinline__ f32x8 frag() const {
    f32x4 a = __builtin_bit_cast(f32x4, r0), b = __builtin_bit_cast(f32x4, r1);
    return f32x8{a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
  }
  __device__ __forceinline__ void set(const float (&v)[8]) {
    r0 = u32x4{__float_as_uint(v[0]), __float_as_uint(v[1]), __float_as_uint(v[2]), __float_as_uint(v[3])};
    r1 = u32x4{__float_as_uint(v[4]), __float_as_uint(v[5]), __float_as_uint(v[6]), __float_as_uint(v[7])};
  }
};

// Transpose an 8x8 block: out[c] element r = in[r] element c.
__device__ __forceinline__ void transpose8x8(const Vec8<bf16> (&in)[8], Vec8<bf16> (&out)[8]) {
#pragma unroll
  for (int c = 0; c < 8; ++c) {
    const int w = c >> 1;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      uint32_t lo = in[2 * i].r[w], hi = in[2 * i + 1].r[w];
      out[c].r[i] = (c & 1) ? ((lo >> 16) | (hi & 0xffff0000u)) : ((lo & 0xffffu) | (hi << 16));
    }
  }
}
__device__ __forceinline__ void transpose8x8(const Vec8<float> (&in)[8], Vec8<float> (&out)[8]) {
#pragma unroll
  for (int c = 0; c < 8; ++c) {
#pragma unroll
    for (int r = 0; r < 8; ++r) {
      uint32_t v = (c < 4) ? in[r].r0[c & 3] : in[r].r1[c & 3];
      if (r < 4) out[c].r0[r & 3] = v; else out[c].r1[r & 3] = v;
    }
  }
}

// Four consecutive elements (8 bytes bf16 / 16 bytes fp32) as a half fragment.
template <typename T> struct Vec4;
template <> struct Vec4<bf16> {
  u32x2 r;
  __device__ __forceinline__ void load(const bf16* p) { r = ld8(p); }
  __device__ __forceinline__ void store(bf16* p) const { st8(p, r); }
  __device__ __forceinline__ float get(int i) const {
    uint32_t w = r[i >> 1];
    return __uint_as_float((i & 1) ? (w & 0xffff0000u) : (w << 16));
  }
  __device__ __forceinline__ void set(const float (&v)[4]) {
    bf16x4 b = {from_f32<bf16>(v[0]), from_f32<bf16>(v[1]), from_f32<bf16>(v[2]), from_f32<bf16>(v[3])};
    r = __builtin_bit_cast(u32x2, b);
  }
};
template <> struct Vec4<float> {
  u32x4 r;
  __device__ __forceinline__ void load(const float* p) { r = ld16(p); }
  __device__ __forceinline__ void store(float* p) const { st16(p, r); }
  __device__ __forceinline__ float get(int i) const { return __uint_as_float(r[i]); }
  __device__ __forceinline__ void set(const float (&v)[4]) {
    r = u32x4{__float_as_uint(v[0]), __float_as_uint(v[1]), __float_as_uint(v[2]), __float_as_uint(v[3])};
  }
};

// Concatenate two half fragments into one eight-slot fragment.
__device__ __forceinline__ bf16x8 join(const Vec4<bf16>& a, const Vec4<bf16>& b) {
  return __builtin_bit_cast(bf16x8, u32x4{a.r[0], a.r[1], b.r[0], b.r[1]});
}
__device__ __forceinline__ f32x8 join(const Vec4<float>& a, const Vec4<float>& b) {
  f32x4 x = __builtin_bit_cast(f32x4, a.r), y = __builtin_bit_cast(f32x4, b.r);
  return f32x8{x[0], x[1], x[2], x[3], y[0], y[1], y[2], y[3]};
}

// Pack eight floats into a fragment of T (bf16: RNE conversion).
__device__ __forceinline__ bf16x8 pack8(const float (&v)[8], bf16*) {
  return bf16x8{from_f32<bf16>(v[0]), from_f32<bf16>(v[1]), from_f32<bf16>(v[2]), from_f32<bf16>(v[3]),
                from_f32<bf16>(v[4]), from_f32<bf16>(v[5]), from_f32<bf16>(v[6]), from_f32<bf16>(v[7])};
}
__device__ __forceinline__ f32x8 pack8(const float (&v)[8], float*) {
  return f32x8{v[0], v[1], v[2], v[3], v[4], v[5], v[6], v[7]};
}

// Wavefront reductions (64 lanes).
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// ---------------------------------------------------------------------------
// Global -> LDS transfers with buffer loads in LDS-DMA mode.
// ---------------------------------------------------------------------------
// Buffer resource: base address, no stride, num_records = bytes, raw
// (untyped) access; reads at or past num_records return zero.
typedef int i32x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ i32x4 buf_rsrc(const void* base, uint32_t bytes) {
  const uint64_t a = reinterpret_cast<uint64_t>(base);
  return i32x4{(int)(uint32_t)a, (int)((a >> 32) & 0xffff), (int)bytes, 0x00020000};
}
// LDS byte address of a __shared__ object (take it once per array and add
// integer offsets; casting derived generic pointers costs a null check).
#define FL_LDS_ADDR(obj) ((uint32_t)(uintptr_t)(__attribute__((address_space(3))) const void*)(obj))
// One instruction: 64 lanes x BYTES (16 or 4) from rs + voff into LDS at
// lds + BYTES * lane (the LDS side ignores per-lane addresses).  Issued as
// inline assembly so that the compiler does not see an LDS write it would
// have to wait for (vmcnt) before every later LDS read: callers wait for a
// stage explicitly, when they publish it with a barrier.
template <int BYTES>
__device__ __forceinline__ void dma_lds(i32x4 rs, uint32_t lds, uint32_t voff) {
  static_assert(BYTES == 16 || BYTES == 4, "dwordx4 or dword");
  const uint32_t m = __builtin_amdgcn_readfirstlane(lds);
  if constexpr (BYTES == 16)
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
                 :
                 : "s"(m), "v"(voff), "s"(rs)
                 : "memory", "m0");
  else
    asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tbuffer_load_dword %1, %2, 0 offen lds"
                 :
                 : "s"(m), "v"(voff), "s"(rs)
                 : "memory", "m0");
}

// Marks a register value as used here.  Values loaded from global memory
// before a loop whose body issues dma_lds() must be settled before the loop:
// otherwise the compiler places its wait for them (vmcnt) inside the body,
// where it would also wait for the in-flight DMA it does not know about.
template <typename T>
__device__ __forceinline__ void settle(T& v) {
  asm volatile("" : "+v"(v));
}

// XOR swizzle of the 8-element chunk index inside an LDS row holding 8
// chunks; spreads both row-wise (fragment reads) and strided (transposed
// writes) access patterns over distinct banks.
__device__ __forceinline__ int swz(int row, int chunk) { return chunk ^ ((row ^ (row >> 3)) & 7); }

}  // namespace flglm
