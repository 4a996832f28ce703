// device.h -- CDNA4 (gfx950) building blocks shared by the prefill kernels:
// 16x16 MFMA tiles for bf16 and fp32 operands, the lane layout of their
// fragments, and conversions.
//
// Tile conventions (one wave64, 16x16 output tile D = A B + C):
//   * accumulator: lane l holds column (l & 15), rows 4*(l >> 4) + e, e = 0..3
//     (an f32x4);
//   * operand fragments cover a k-block of 32: lane l feeds row (A) or column
//     (B) (l & 15) with 8 values; lane group grp = l >> 4 supplies 8 of the 32
//     k indices.  A and B of one product must agree on which logical k index
//     each (grp, j) slot carries; the hardware's own slot order never matters.
//   * two slot maps are used:
//       contiguous   kc(grp, j) = 8*grp + j            -- both operands read
//                    from memory: one 16-byte load per lane (load_frag);
//       accumulator  kmap(grp, j) = 4*grp + j (j < 4), 16 + 4*grp + j - 4 (j >= 4)
//                    -- the map under which an accumulator pair (rows 0-15
//                    tile, rows 16-31 tile) IS the B fragment of a k-block over
//                    those 32 rows, lane for lane (frag_from_acc): a result
//                    feeds the next product with no cross-lane movement.  The
//                    partner A operand of such a product is stored
//                    "kmap-permuted": inside every 32-block, position 8*grp + j
//                    holds logical index kmap(grp, j).  It is then read with
//                    the same contiguous 16-byte load_frag.
// bf16 operands use v_mfma_f32_16x16x32_bf16 (one instruction per k-block);
// fp32 operands use v_mfma_f32_16x16x4_f32 (eight instructions per k-block,
// step j contracting the four values j of the four lane groups).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace hagdn {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x8 __attribute__((ext_vector_type(8)));
// 16 raw bytes as a native vector: unlike HIP's union-based uint4 it stays in
// registers when held in arrays.
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef uint16_t bf16_t;  // bf16 storage

__device__ __forceinline__ int lane_id() { return threadIdx.x & 63; }

// --------------------------------------------------------------- conversions
__device__ __forceinline__ float bf16_to_f32(bf16_t x) {
  return __uint_as_float(((uint32_t)x) << 16);
}
// Round to nearest even (the hardware conversion on gfx950).
__device__ __forceinline__ bf16_t f32_to_bf16(float x) {
  __bf16 b = (__bf16)x;
  return __builtin_bit_cast(bf16_t, b);
}

template <typename T> struct Elt;
template <> struct Elt<bf16_t> {
  using frag = bf16x8;
  __device__ static float to_f32(bf16_t x) { return bf16_to_f32(x); }
  __device__ static bf16_t from_f32(float x) { return f32_to_bf16(x); }
};
template <> struct Elt<float> {
  using frag = f32x8;
  __device__ static float to_f32(float x) { return x; }
  __device__ static float from_f32(float x) { return x; }
};

template <typename T> using Frag = typename Elt<T>::frag;

// logical k index of slot j of lane group grp under the accumulator map
__device__ __forceinline__ constexpr int kmap(int grp, int j) {
  return j < 4 ? 4 * grp + j : 12 + 4 * grp + j;
}
// position inside a kmap-permuted 32-block of logical index i (0..31)
__device__ __forceinline__ constexpr int kmap_pos(int i) {
  return i < 16 ? 8 * (i >> 2) + (i & 3) : 8 * ((i - 16) >> 2) + 4 + (i & 3);
}

// d_v column held by column j (0..15) of state tile n.  Tile pairs (2p, 2p+1)
// interleave in groups of four, so the eight output values a lane computes
// for tiles 2p and 2p+1 (rows 4grp + e of each) are eight consecutive columns
// 32p + 8grp + 0..7: one 16-byte store.  A bijection of [0, 32p + 32).
__device__ __forceinline__ constexpr int dv_of(int n, int j) {
  return 32 * (n >> 1) + 8 * (j >> 2) + 4 * (n & 1) + (j & 3);
}

// ------------------------------------------------------------ 4-element I/O
// Four consecutive elements as fp32 (8-byte load for bf16, 16-byte for fp32).
__device__ __forceinline__ f32x4 load4(const bf16_t *p) {
  uint2 u = *reinterpret_cast<const uint2 *>(p);
  f32x4 r;
  r[0] = __uint_as_float(u.x << 16);
  r[1] = __uint_as_float(u.x & 0xffff0000u);
  r[2] = __uint_as_float(u.y << 16);
  r[3] = __uint_as_float(u.y & 0xffff0000u);
  return r;
}
__device__ __forceinline__ f32x4 load4(const float *p) {
  return *reinterpret_cast<const f32x4 *>(p);
}
__device__ __forceinline__ void store4(bf16_t *p, f32x4 v) {
  uint2 u;
  u.x = (uint32_t)f32_to_bf16(v[0]) | ((uint32_t)f32_to_bf16(v[1]) << 16);
  u.y = (uint32_t)f32_to_bf16(v[2]) | ((uint32_t)f32_to_bf16(v[3]) << 16);
  *reinterpret_cast<uint2 *>(p) = u;
}
__device__ __forceinline__ void store4(float *p, f32x4 v) {
  *reinterpret_cast<f32x4 *>(p) = v;
}

// Eight consecutive elements from two accumulator quads (one 16-byte store
// for bf16, two for fp32).
__device__ __forceinline__ void store8(bf16_t *p, f32x4 lo, f32x4 hi);
__device__ __forceinline__ void store8(float *p, f32x4 lo, f32x4 hi) {
  *reinterpret_cast<f32x4 *>(p) = lo;
  *reinterpret_cast<f32x4 *>(p + 4) = hi;
}

// ---------------------------------------------------- 16-byte vector access
// A uint4 holds 8 bf16 or 4 fp32 elements; element j (compile-time after
// unrolling) read as fp32, read raw, or packed from fp32 with rounding.
__device__ __forceinline__ uint32_t word(uint4 u, int i) {
  return i == 0 ? u.x : i == 1 ? u.y : i == 2 ? u.z : u.w;
}
template <typename T> struct Vec16;
template <> struct Vec16<bf16_t> {
  static constexpr int N = 8;
  __device__ static float get(uint4 u, int j) {
    const uint32_t w = word(u, j >> 1);
    return __uint_as_float((j & 1) ? (w & 0xffff0000u) : (w << 16));
  }
  __device__ static bf16_t raw(uint4 u, int j) {
    const uint32_t w = word(u, j >> 1);
    return (bf16_t)((j & 1) ? (w >> 16) : (w & 0xffffu));
  }
  __device__ static uint4 pack(const float (&x)[8]) {
    uint32_t w[4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
      w[i] = (uint32_t)f32_to_bf16(x[2 * i]) | ((uint32_t)f32_to_bf16(x[2 * i + 1]) << 16);
    return make_uint4(w[0], w[1], w[2], w[3]);
  }
};
template <> struct Vec16<float> {
  static constexpr int N = 4;
  __device__ static float get(uint4 u, int j) { return __uint_as_float(word(u, j)); }
  __device__ static float raw(uint4 u, int j) { return __uint_as_float(word(u, j)); }
  __device__ static uint4 pack(const float (&x)[4]) {
    return make_uint4(__float_as_uint(x[0]), __float_as_uint(x[1]), __float_as_uint(x[2]),
                      __float_as_uint(x[3]));
  }
};

// ------------------------------------------------------------- fragments
// Fragment of the 32-block at p: lane group grp reads elements [8*grp, 8*grp + 8)
// (one 16-byte load for bf16).  Logical order under the contiguous map, or
// kmap order when the block is stored kmap-permuted.
__device__ __forceinline__ bf16x8 load_frag(const bf16_t *p, int grp) {
  return __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4 *>(p + 8 * grp));
}
__device__ __forceinline__ f32x8 load_frag(const float *p, int grp) {
  f32x4 a = *reinterpret_cast<const f32x4 *>(p + 8 * grp);
  f32x4 b = *reinterpret_cast<const f32x4 *>(p + 8 * grp + 4);
  f32x8 r;
  r[0] = a[0]; r[1] = a[1]; r[2] = a[2]; r[3] = a[3];
  r[4] = b[0]; r[5] = b[1]; r[6] = b[2]; r[7] = b[3];
  return r;
}
// Contiguous-map logical k index of slot j of lane group grp.
__device__ __forceinline__ constexpr int kc(int grp, int j) { return 8 * grp + j; }

// Fragment from eight fp32 values (in kmap order), rounded to the operand type.
template <typename T> __device__ __forceinline__ Frag<T> make_frag(const float (&x)[8]);
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
template <> __device__ __forceinline__ bf16x8 make_frag<bf16_t>(const float (&x)[8]) {
  // two packed conversions per 4 values (v_cvt_pk_bf16_f32), no repacking
  const f32x4 lo = {x[0], x[1], x[2], x[3]}, hi = {x[4], x[5], x[6], x[7]};
  const bf16x4 a = __builtin_convertvector(lo, bf16x4), b = __builtin_convertvector(hi, bf16x4);
  return __builtin_shufflevector(a, b, 0, 1, 2, 3, 4, 5, 6, 7);
}
template <> __device__ __forceinline__ f32x8 make_frag<float>(const float (&x)[8]) {
  f32x8 r;
#pragma unroll
  for (int j = 0; j < 8; ++j) r[j] = x[j];
  return r;
}

// B fragment over 32 rows from two accumulator tiles (rows 0-15, rows 16-31).
template <typename T> __device__ __forceinline__ Frag<T> frag_from_acc(f32x4 lo, f32x4 hi);
template <> __device__ __forceinline__ bf16x8 frag_from_acc<bf16_t>(f32x4 lo, f32x4 hi) {
  const bf16x4 a = __builtin_convertvector(lo, bf16x4), b = __builtin_convertvector(hi, bf16x4);
  return __builtin_shufflevector(a, b, 0, 1, 2, 3, 4, 5, 6, 7);
}
template <> __device__ __forceinline__ f32x8 frag_from_acc<float>(f32x4 lo, f32x4 hi) {
  return __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
}

// Fragment-order ("swizzled") blocks: a 16x32 operand block stored as 64 lanes
// x 8 consecutive elements, lane-major, exactly as the MFMA fragment sits in a
// wave.  A wave reads or writes one such block as a single contiguous 1 KiB
// (bf16) run.  load_frag_at / store_frag_at address this lane's 8 elements.
__device__ __forceinline__ bf16x8 load_frag_at(const bf16_t *p) {
  return __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4 *>(p));
}
__device__ __forceinline__ f32x8 load_frag_at(const float *p) {
  const f32x4 a = *reinterpret_cast<const f32x4 *>(p);
  const f32x4 b = *reinterpret_cast<const f32x4 *>(p + 4);
  return __builtin_shufflevector(a, b, 0, 1, 2, 3, 4, 5, 6, 7);
}
__device__ __forceinline__ void store_frag_at(bf16_t *p, bf16x8 f) {
  *reinterpret_cast<uint4 *>(p) = __builtin_bit_cast(uint4, f);
}
__device__ __forceinline__ void store_frag_at(float *p, f32x8 f) {
  *reinterpret_cast<f32x4 *>(p) = __builtin_shufflevector(f, f, 0, 1, 2, 3);
  *reinterpret_cast<f32x4 *>(p + 4) = __builtin_shufflevector(f, f, 4, 5, 6, 7);
}

__device__ __forceinline__ void store8(bf16_t *p, f32x4 lo, f32x4 hi) {
  *reinterpret_cast<uint4 *>(p) = __builtin_bit_cast(uint4, frag_from_acc<bf16_t>(lo, hi));
}

// Store a fragment where load_frag would read it: 8 elements at p + 8*grp.
__device__ __forceinline__ void store_frag(bf16_t *p, bf16x8 f, int grp) {
  *reinterpret_cast<uint4 *>(p + 8 * grp) = __builtin_bit_cast(uint4, f);
}
__device__ __forceinline__ void store_frag(float *p, f32x8 f, int grp) {
  *reinterpret_cast<f32x4 *>(p + 8 * grp) = __builtin_shufflevector(f, f, 0, 1, 2, 3);
  *reinterpret_cast<f32x4 *>(p + 8 * grp + 4) = __builtin_shufflevector(f, f, 4, 5, 6, 7);
}

// Element j of a fragment as fp32 (exact).
__device__ __forceinline__ float frag_elem(bf16x8 f, int j) { return (float)f[j]; }
__device__ __forceinline__ float frag_elem(f32x8 f, int j) { return f[j]; }

template <typename T> __device__ __forceinline__ Frag<T> zero_frag() {
  float x[8] = {0, 0, 0, 0, 0, 0, 0, 0};
  return make_frag<T>(x);
}

// --------------------------------------------------------------------- MFMA
__device__ __forceinline__ f32x4 mma(f32x4 acc, bf16x8 a, bf16x8 b) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, acc, 0, 0, 0);
}
__device__ __forceinline__ f32x4 mma(f32x4 acc, f32x8 a, f32x8 b) {
#pragma unroll
  for (int j = 0; j < 8; ++j) acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a[j], b[j], acc, 0, 0, 0);
  return acc;
}

// ------------------------------------------------ input preprocessing maps
// Raw projection -> log-gate: -softplus(x) = -(max(x, 0) + log(1 + e^-|x|)),
// the form in which the exponential cannot overflow.
__device__ __forceinline__ float neg_softplus(float x) {
  return -(fmaxf(x, 0.f) + log1pf(expf(-fabsf(x))));
}
// Raw projection -> write strength in (0, 1).
__device__ __forceinline__ float sigmoid(float x) { return 1.f / (1.f + expf(-x)); }
// Factor that L2-normalises a vector with squared norm ss (norm floored at 1e-6).
__device__ __forceinline__ float inv_l2(float ss) { return 1.f / fmaxf(sqrtf(ss), 1e-6f); }
// Sum over the 64 lanes of a wave, every lane receives it.
__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) x += __shfl_xor(x, off);
  return x;
}

__device__ __forceinline__ f32x4 zero4() {
  f32x4 z = {0.f, 0.f, 0.f, 0.f};
  return z;
}

}  // namespace hagdn
