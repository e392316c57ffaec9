// Shared device helpers for the gfx950 kernels: bf16 storage conversion,
// MFMA operand vector types, wave-level utilities and launch error plumbing.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stddef.h>

namespace lat {

typedef uint16_t bf16_t;  // bf16 in memory: the upper 16 bits of an fp32

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

enum DType { DT_F32 = 0, DT_BF16 = 1 };

constexpr int WAVE = 64;

__host__ __device__ inline float bf2f(bf16_t h) {
  union { uint32_t u; float f; } v;
  v.u = (uint32_t)h << 16;
  return v.f;
}

// fp32 -> bf16, round to nearest even; NaN stays NaN.  On the GPU this is the
// hardware conversion (v_cvt_pk_bf16_f32 on gfx950); the host keeps the
// bit-level rounding.
__host__ __device__ inline bf16_t f2bf(float f) {
#if defined(__HIP_DEVICE_COMPILE__)
  return __builtin_bit_cast(bf16_t, (__bf16)f);
#else
  union { uint32_t u; float f; } v;
  v.f = f;
  uint32_t u = v.u;
  if ((u & 0x7fffffffu) > 0x7f800000u) return (bf16_t)((u >> 16) | 0x40);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (bf16_t)(u >> 16);
#endif
}

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));

// two fp32 -> two bf16 in one 32-bit word (a in the low half), one instruction
__device__ inline uint32_t pack_bf2(float a, float b) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2_t{a, b}, bf16x2_t));
}

template <typename T> struct Elt;
template <> struct Elt<float> {
  __device__ static inline float load(const float* p) { return *p; }
  __device__ static inline void store(float* p, float v) { *p = v; }
};
template <> struct Elt<bf16_t> {
  __device__ static inline float load(const bf16_t* p) { return bf2f(*p); }
  __device__ static inline void store(bf16_t* p, float v) { *p = f2bf(v); }
};

template <typename T> __device__ inline float ld(const T* p) { return Elt<T>::load(p); }
// value of v after a round trip through storage type T
template <typename T> __device__ inline float ld_round(float v);
template <> __device__ inline float ld_round<float>(float v) { return v; }
template <> __device__ inline float ld_round<bf16_t>(float v) { return bf2f(f2bf(v)); }
template <typename T> __device__ inline void st(T* p, float v) { Elt<T>::store(p, v); }

// 16-byte vector <-> fp32 lanes.  A 16-byte vector holds 8 bf16 or 4 fp32.
template <typename T> struct Vec16;
template <> struct Vec16<bf16_t> {
  static constexpr int N = 8;
  __device__ static inline void unpack(const u32x4& v, float* o) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      o[2 * i] = __uint_as_float(v[i] << 16);
      o[2 * i + 1] = __uint_as_float(v[i] & 0xffff0000u);
    }
  }
  __device__ static inline u32x4 pack(const float* o) {
    u32x4 v;
#pragma unroll
    for (int i = 0; i < 4; ++i) v[i] = pack_bf2(o[2 * i], o[2 * i + 1]);
    return v;
  }
};
template <> struct Vec16<float> {
  static constexpr int N = 4;
  __device__ static inline void unpack(const u32x4& v, float* o) {
#pragma unroll
    for (int i = 0; i < 4; ++i) o[i] = __uint_as_float(v[i]);
  }
  __device__ static inline u32x4 pack(const float* o) {
    u32x4 v;
#pragma unroll
    for (int i = 0; i < 4; ++i) v[i] = __float_as_uint(o[i]);
    return v;
  }
};

__device__ inline u32x4 ldg16(const void* p) { return *reinterpret_cast<const u32x4*>(p); }
__device__ inline void stg16(void* p, const u32x4& v) { *reinterpret_cast<u32x4*>(p) = v; }

inline int cdiv(int64_t a, int64_t b) { return (int)((a + b - 1) / b); }

// MI355X has 8 XCDs, each with its own L2; consecutive workgroup ids are
// dealt to the XCDs round-robin.  xcd_block() renumbers the linear block id
// so that each XCD walks one contiguous share of [0, nblocks): work items
// that are neighbours in the renumbered order share one L2.  A bijection on
// [0, nblocks).
constexpr int NUM_XCD = 8;

// Word 3 of a raw (untyped, unswizzled) buffer resource on gfx9-family GPUs.
constexpr int BUF_RSRC_WORD3 = 0x00020000;
// Cache-policy operand of a buffer access: non-temporal (the nt bit of gfx94x/gfx950).
constexpr int BUF_NT = 2;
__device__ inline int xcd_block(int bid, int nblocks) {
  const int x = bid % NUM_XCD, i = bid / NUM_XCD;
  const int q = nblocks / NUM_XCD, r = nblocks % NUM_XCD;
  return x * q + (x < r ? x : r) + i;
}

}  // namespace lat

// Host-side error plumbing shared by the launchers.
namespace lat {
void set_error(const char* fmt, ...);
}

#define LAT_HIP_CHECK(expr)                                                  \
  do {                                                                       \
    hipError_t e_ = (expr);                                                  \
    if (e_ != hipSuccess) {                                                  \
      ::lat::set_error("%s: %s (%s:%d)", #expr, hipGetErrorString(e_),       \
                       __FILE__, __LINE__);                                  \
      return e_;                                                             \
    }                                                                        \
  } while (0)

#define LAT_LAUNCH_CHECK() LAT_HIP_CHECK(hipGetLastError())
