// Helpers shared by the gfx950 kernels: storage types, bf16 conversion,
// vector loads/stores, wave64 reductions and MFMA operand types (device side),
// and the per-device dynamic-LDS attribute (host side).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <atomic>

namespace merak {

typedef uint16_t bf16_t;  // bf16 storage (bit pattern)

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));  // 16-byte register
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));

// bf16 <-> fp32.  The narrowing rounds to nearest, ties to even (gfx950 has a
// hardware instruction for it).
__device__ __forceinline__ float bf2f(bf16_t v) { return __uint_as_float(((uint32_t)v) << 16); }
__device__ __forceinline__ bf16_t f2bf(float f) {
  __bf16 b = (__bf16)f;
  return __builtin_bit_cast(uint16_t, b);
}

// Element traits: bf16 storage (fp32 math) or fp32 check mode.
template <typename T> struct Elem;
template <> struct Elem<bf16_t> {
  static __device__ __forceinline__ float to_f(bf16_t v) { return bf2f(v); }
  static __device__ __forceinline__ bf16_t from_f(float f) { return f2bf(f); }
};
template <> struct Elem<float> {
  static __device__ __forceinline__ float to_f(float v) { return v; }
  static __device__ __forceinline__ float from_f(float f) { return f; }
};

// Four / eight consecutive elements <-> float[4] / float[8] (native vector
// types, so values stay in registers).
__device__ __forceinline__ void load4(const bf16_t* p, float v[4]) {
  u32x2_t r = *reinterpret_cast<const u32x2_t*>(p);
  v[0] = __uint_as_float(r[0] << 16);
  v[1] = __uint_as_float(r[0] & 0xffff0000u);
  v[2] = __uint_as_float(r[1] << 16);
  v[3] = __uint_as_float(r[1] & 0xffff0000u);
}
__device__ __forceinline__ void load4(const float* p, float v[4]) {
  f32x4_t r = *reinterpret_cast<const f32x4_t*>(p);
  v[0] = r[0]; v[1] = r[1]; v[2] = r[2]; v[3] = r[3];
}
// Two values narrowed by one packed conversion instruction (converting them
// one at a time costs two conversions plus a shift and an OR).
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_t{lo, hi}, bf16x2_t));
}
__device__ __forceinline__ void store4(bf16_t* p, const float v[4]) {
  *reinterpret_cast<u32x2_t*>(p) = u32x2_t{pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3])};
}
__device__ __forceinline__ void store4(float* p, const float v[4]) {
  *reinterpret_cast<f32x4_t*>(p) = f32x4_t{v[0], v[1], v[2], v[3]};
}
__device__ __forceinline__ void unpack8(const u32x4_t r, float v[8]) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    v[2 * i] = __uint_as_float(r[i] << 16);
    v[2 * i + 1] = __uint_as_float(r[i] & 0xffff0000u);
  }
}
__device__ __forceinline__ void load8(const bf16_t* p, float v[8]) {
  unpack8(*reinterpret_cast<const u32x4_t*>(p), v);
}
__device__ __forceinline__ void load8(const float* p, float v[8]) {
  f32x4_t a = reinterpret_cast<const f32x4_t*>(p)[0];
  f32x4_t b = reinterpret_cast<const f32x4_t*>(p)[1];
  v[0] = a[0]; v[1] = a[1]; v[2] = a[2]; v[3] = a[3];
  v[4] = b[0]; v[5] = b[1]; v[6] = b[2]; v[7] = b[3];
}
__device__ __forceinline__ void store8(bf16_t* p, const float v[8]) {
  *reinterpret_cast<u32x4_t*>(p) = u32x4_t{pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3]),
                                           pack_bf16x2(v[4], v[5]), pack_bf16x2(v[6], v[7])};
}
__device__ __forceinline__ void store8(float* p, const float v[8]) {
  reinterpret_cast<f32x4_t*>(p)[0] = f32x4_t{v[0], v[1], v[2], v[3]};
  reinterpret_cast<f32x4_t*>(p)[1] = f32x4_t{v[4], v[5], v[6], v[7]};
}

// Wave64 reductions (butterfly over all 64 lanes; every lane gets the result).
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v = fmaxf(v, __shfl_xor(v, off, 64));
  return v;
}

// GeLU, tanh form, and its derivative, written with s = sigmoid(2z) =
// 1 / (1 + exp(-2z)), z = sqrt(2/pi) (u + 0.044715 u^3): since
// 1 + tanh(z) = 2 s and 1 - tanh(z)^2 = 4 s (1 - s),
//   gelu(u)  = u s,
//   gelu'(u) = s + 2 u s (1 - s) sqrt(2/pi) (1 + 3 * 0.044715 u^2).
// One exponential and one hardware reciprocal (about 1 ulp) per element; both
// saturate correctly for large |u| (exp -> inf gives s = 0, exp -> 0 gives 1).
constexpr float kGeluC = 0.7978845608028654f;  // sqrt(2/pi)
constexpr float kGeluA = 0.044715f;
__device__ __forceinline__ float gelu_sigmoid(float u) {
  const float z2 = 2.0f * kGeluC * (u + kGeluA * u * u * u);
  return __builtin_amdgcn_rcpf(1.0f + __expf(-z2));
}
__device__ __forceinline__ float gelu_f(float u) { return u * gelu_sigmoid(u); }
__device__ __forceinline__ float gelu_grad_f(float u) {
  const float s = gelu_sigmoid(u);
  return s + 2.0f * u * s * (1.0f - s) * kGeluC * (1.0f + 3.0f * kGeluA * u * u);
}

// Host side: allow a kernel `bytes` of dynamic LDS beyond the default limit on
// the current device.  The attribute is held per device, so it is set once for
// each device the kernel runs on (bit d of `done`; devices past 63 set it on
// every launch).  The call is idempotent, so host threads racing on a first
// launch are harmless.
inline hipError_t allow_dynamic_lds(const void* kern, size_t bytes, std::atomic<uint64_t>& done) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  const uint64_t bit = dev >= 0 && dev < 64 ? (uint64_t)1 << dev : 0;
  if (bit && (done.load(std::memory_order_acquire) & bit)) return hipSuccess;
  e = hipFuncSetAttribute(kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
  if (e == hipSuccess && bit) done.fetch_or(bit, std::memory_order_acq_rel);
  return e;
}

}  // namespace merak
