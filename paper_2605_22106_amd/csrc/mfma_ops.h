// MFMA operand helpers shared by the score and decode kernels (gfx950).
//
// Both kernels use the 16x16 MFMA family.  For a 16 x 16 output tile a lane
// l supplies row (l % 16) of the A operand and column (l % 16) of the B operand,
// each for the k-slice owned by lane group l / 16, and receives rows
// 4 * (l / 16) + e (e < 4) of output column l % 16.  Because A and B take their
// k-slice from the same lane group, the reduction dimension may be permuted
// freely as long as both operands use the same permutation.
#pragma once

#include <hip/hip_runtime.h>

namespace arbor {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

template <class T>
struct Op;

// bf16 inputs: v_mfma_f32_16x16x32_bf16, 8 elements of k per lane per step.
template <>
struct Op<__bf16> {
  typedef bf16x8 reg;
  static constexpr int kPerStep = 8;
  static __device__ __forceinline__ f32x4 mma(reg a, reg b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
  }
  static __device__ __forceinline__ reg load(const __bf16 *p) {
    return *reinterpret_cast<const bf16x8 *>(p);
  }
  static __device__ __forceinline__ reg zero() {
    reg r;
#pragma unroll
    for (int e = 0; e < 8; ++e) r[e] = (__bf16)0.0f;
    return r;
  }
};

// fp32 inputs: v_mfma_f32_16x16x4_f32, one element of k per lane per step.
template <>
struct Op<float> {
  typedef float reg;
  static constexpr int kPerStep = 1;
  static __device__ __forceinline__ f32x4 mma(reg a, reg b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
  }
  static __device__ __forceinline__ reg load(const float *p) { return *p; }
  static __device__ __forceinline__ reg zero() { return 0.0f; }
};

// Column of head_dim that lane group g4 supplies at MFMA k-step ks.  Both
// operands of a dot product use the same map, so the result is unchanged; it
// makes the four lane groups of one k-step read consecutive 16-byte pieces of
// a row, so a 16-row fragment load touches 64 contiguous bytes of each row.
template <class T>
__device__ __forceinline__ int frag_col(int ks, int g4) {
  constexpr int VEC = 16 / (int)sizeof(T);          // elements per 16 bytes
  constexpr int SPV = VEC / Op<T>::kPerStep;        // k-steps per 16 bytes
  return (ks / SPV) * 4 * VEC + g4 * VEC + (ks % SPV) * Op<T>::kPerStep;
}

// fp32 MFMA 16x16x4 (A, B scalars per lane), used for P V with fp32 P.
__device__ __forceinline__ f32x4 mma_f32(float a, float b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

// n consecutive elements of T widened to float.
template <class T, int NC>
__device__ __forceinline__ void load_row_f32(const T *p, float (&out)[NC]);

template <>
__device__ __forceinline__ void load_row_f32<__bf16, 8>(const __bf16 *p, float (&out)[8]) {
  const bf16x8 v = *reinterpret_cast<const bf16x8 *>(p);
#pragma unroll
  for (int e = 0; e < 8; ++e) out[e] = (float)v[e];
}
template <>
__device__ __forceinline__ void load_row_f32<__bf16, 4>(const __bf16 *p, float (&out)[4]) {
  typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
  const bf16x4 v = *reinterpret_cast<const bf16x4 *>(p);
#pragma unroll
  for (int e = 0; e < 4; ++e) out[e] = (float)v[e];
}
template <>
__device__ __forceinline__ void load_row_f32<float, 8>(const float *p, float (&out)[8]) {
  const float4 a = *reinterpret_cast<const float4 *>(p);
  const float4 b = *reinterpret_cast<const float4 *>(p + 4);
  out[0] = a.x; out[1] = a.y; out[2] = a.z; out[3] = a.w;
  out[4] = b.x; out[5] = b.y; out[6] = b.z; out[7] = b.w;
}
template <>
__device__ __forceinline__ void load_row_f32<float, 4>(const float *p, float (&out)[4]) {
  const float4 a = *reinterpret_cast<const float4 *>(p);
  out[0] = a.x; out[1] = a.y; out[2] = a.z; out[3] = a.w;
}

}  // namespace arbor
