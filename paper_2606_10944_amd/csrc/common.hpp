// Device-side building blocks shared by the thinning kernels (gfx950 / CDNA4).
//
// Row fragments.  A 64-lane wavefront covers 16 rows of a d-wide matrix:
// lane l holds row (l % 16) and, in its v-th 16-byte word, the row's word
// 4v + l/16.  One load instruction therefore reads 64 contiguous bytes of
// each row.  The same lane layout serves as the A operand (rows = M) and as
// the B operand (rows = N) of the 16x16 MFMA instructions: within one
// instruction, lane group l/16 feeds the same k-slots to A and B, so the
// product of two fragments is the matrix of row dot products <row_m, row_n>
// whatever the internal k order is.
//
// 16x16 MFMA outputs: lane l holds D[4*(l/16) + i][l % 16], i = 0..3.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace thin {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float floatx4_t __attribute__((ext_vector_type(4)));
// Native 16-byte vector: arrays of it stay in registers where arrays of the
// HIP uint4 class can be demoted to scratch memory.
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

struct bf16_t {
  uint16_t bits;
};

template <typename T>
struct Elem;

template <>
struct Elem<float> {
  static constexpr int bytes = 4;
  static constexpr uint32_t sign_mask = 0x80000000u;
};
template <>
struct Elem<bf16_t> {
  static constexpr int bytes = 2;
  static constexpr uint32_t sign_mask = 0x80008000u;
};

// Number of 16-byte words a lane holds for a d-wide row of T.
template <typename T, int D>
struct Frag {
  static constexpr int elems = D / 4;
  static constexpr int NV = elems * Elem<T>::bytes / 16;
  static_assert(NV >= 1, "row quarter must be at least 16 bytes");
};

__device__ __forceinline__ float bf16_to_float(uint16_t b) {
  return __uint_as_float(((uint32_t)b) << 16);
}

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

// Two floats to two bf16 (round to nearest even) in one word, a in the low
// half: one packed conversion instruction on gfx950.
__device__ __forceinline__ uint32_t cvt_pk_bf16(float a, float b) {
  const bf16x2_t v = {(__bf16)a, (__bf16)b};
  return __builtin_bit_cast(uint32_t, v);
}

// Eight values (probabilities of the P V product) as bf16 high parts and the
// bf16 rounding of what each high part leaves: hi + lo carries about 16
// significant bits of each value, so two bf16 MFMAs give P V to about the
// accuracy of float32 P.
__device__ __forceinline__ void split_bf16x8(const float* p, bf16x8_t& hi, bf16x8_t& lo) {
  uint32_t h[4], l[4];
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    h[k] = cvt_pk_bf16(p[2 * k], p[2 * k + 1]);
    l[k] = cvt_pk_bf16(p[2 * k] - __uint_as_float(h[k] << 16),
                       p[2 * k + 1] - __uint_as_float(h[k] & 0xffff0000u));
  }
  hi = __builtin_bit_cast(bf16x8_t, make_uint4(h[0], h[1], h[2], h[3]));
  lo = __builtin_bit_cast(bf16x8_t, make_uint4(l[0], l[1], l[2], l[3]));
}

// acc += A_frag x B_frag over one row fragment.
template <typename T, int D>
__device__ __forceinline__ floatx4_t mma_rows(const uint4* a, const uint4* b, floatx4_t acc);

template <>
__device__ __forceinline__ floatx4_t mma_rows<bf16_t, 32>(const uint4* a, const uint4* b,
                                                         floatx4_t acc) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a[0]),
                                                 __builtin_bit_cast(bf16x8_t, b[0]), acc, 0, 0, 0);
}
template <>
__device__ __forceinline__ floatx4_t mma_rows<bf16_t, 64>(const uint4* a, const uint4* b,
                                                         floatx4_t acc) {
#pragma unroll
  for (int v = 0; v < 2; ++v)
    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a[v]),
                                                  __builtin_bit_cast(bf16x8_t, b[v]), acc, 0, 0, 0);
  return acc;
}
template <>
__device__ __forceinline__ floatx4_t mma_rows<bf16_t, 128>(const uint4* a, const uint4* b,
                                                          floatx4_t acc) {
#pragma unroll
  for (int v = 0; v < 4; ++v)
    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a[v]),
                                                  __builtin_bit_cast(bf16x8_t, b[v]), acc, 0, 0, 0);
  return acc;
}

template <int NV>
__device__ __forceinline__ floatx4_t mma_rows_f32(const uint4* a, const uint4* b, floatx4_t acc) {
#pragma unroll
  for (int v = 0; v < NV; ++v) {
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a[v].x), __uint_as_float(b[v].x), acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a[v].y), __uint_as_float(b[v].y), acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a[v].z), __uint_as_float(b[v].z), acc, 0, 0, 0);
    acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a[v].w), __uint_as_float(b[v].w), acc, 0, 0, 0);
  }
  return acc;
}
template <>
__device__ __forceinline__ floatx4_t mma_rows<float, 32>(const uint4* a, const uint4* b, floatx4_t acc) {
  return mma_rows_f32<2>(a, b, acc);
}
template <>
__device__ __forceinline__ floatx4_t mma_rows<float, 64>(const uint4* a, const uint4* b, floatx4_t acc) {
  return mma_rows_f32<4>(a, b, acc);
}
template <>
__device__ __forceinline__ floatx4_t mma_rows<float, 128>(const uint4* a, const uint4* b, floatx4_t acc) {
  return mma_rows_f32<8>(a, b, acc);
}

// acc += A_word x B_word for one 16-byte word of the row fragments (one
// k-chunk): 16x16x32 bf16 (one MFMA) or 16x16x4 f32 (four MFMAs).
template <typename T>
__device__ __forceinline__ floatx4_t mma_word(const uint4& a, const uint4& b, floatx4_t acc);

template <>
__device__ __forceinline__ floatx4_t mma_word<bf16_t>(const uint4& a, const uint4& b, floatx4_t acc) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                 __builtin_bit_cast(bf16x8_t, b), acc, 0, 0, 0);
}
template <>
__device__ __forceinline__ floatx4_t mma_word<float>(const uint4& a, const uint4& b, floatx4_t acc) {
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.x), __uint_as_float(b.x), acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.y), __uint_as_float(b.y), acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.z), __uint_as_float(b.z), acc, 0, 0, 0);
  acc = __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.w), __uint_as_float(b.w), acc, 0, 0, 0);
  return acc;
}

// acc += A_word x B_word using only k-slot 0 of lane group 0 (one MFMA).
template <typename T>
__device__ __forceinline__ floatx4_t mma_aug(const uint4& a, const uint4& b, floatx4_t acc);

template <>
__device__ __forceinline__ floatx4_t mma_aug<bf16_t>(const uint4& a, const uint4& b, floatx4_t acc) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                 __builtin_bit_cast(bf16x8_t, b), acc, 0, 0, 0);
}
template <>
__device__ __forceinline__ floatx4_t mma_aug<float>(const uint4& a, const uint4& b, floatx4_t acc) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(__uint_as_float(a.x), __uint_as_float(b.x), acc, 0, 0, 0);
}

// Load this lane's quarter of row `row` (d columns of T) or zeros if !valid.
template <typename T, int D>
__device__ __forceinline__ void load_frag(const T* base, int64_t row, int g, bool valid, uint4* out) {
  constexpr int NV = Frag<T, D>::NV;
  if (valid) {
    const uint4* p = reinterpret_cast<const uint4*>(base + row * D);
#pragma unroll
    for (int v = 0; v < NV; ++v) out[v] = p[4 * v + g];
  } else {
#pragma unroll
    for (int v = 0; v < NV; ++v) out[v] = make_uint4(0, 0, 0, 0);
  }
}

template <typename T>
__device__ __forceinline__ float elem_to_float(const uint4* w, int e);

template <>
__device__ __forceinline__ float elem_to_float<float>(const uint4* w, int e) {
  const uint32_t* u = reinterpret_cast<const uint32_t*>(w);
  return __uint_as_float(u[e]);
}
template <>
__device__ __forceinline__ float elem_to_float<bf16_t>(const uint4* w, int e) {
  const uint16_t* u = reinterpret_cast<const uint16_t*>(w);
  return bf16_to_float(u[e]);
}

}  // namespace thin
