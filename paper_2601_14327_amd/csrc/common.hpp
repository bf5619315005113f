// Internal helpers shared by the gfx950 kernels of the LAEP MoE library.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace laep {

// ---------------------------------------------------------------------------
// Types
// ---------------------------------------------------------------------------
typedef uint16_t bf16_t;  // raw bf16 bits (IEEE binary32 upper half)

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));

constexpr int kWave = 64;

// ---------------------------------------------------------------------------
// bf16 <-> fp32.  bf16 keeps the sign, the 8 exponent bits and the top 7
// fraction bits of binary32.  Narrowing uses gfx950's v_cvt_pk_bf16_f32
// (round to nearest, ties to even; NaN stays NaN), which the compiler emits
// for a float -> __bf16 conversion; it is branch-free.
// ---------------------------------------------------------------------------
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));

__device__ __forceinline__ float bf16_to_f32(uint32_t b) {
  return __uint_as_float(b << 16);
}

// two floats -> packed bf16x2 (lo in bits 0..15)
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  const bf16x2_t v = {(__bf16)lo, (__bf16)hi};
  return __builtin_bit_cast(uint32_t, v);
}

__device__ __forceinline__ uint32_t f32_to_bf16(float f) { return pack_bf16x2(f, 0.0f) & 0xFFFFu; }

__device__ __forceinline__ float lo_bf16(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float hi_bf16(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// ---------------------------------------------------------------------------
// Streaming (non-temporal) 16-byte accesses for data touched once: measured
// on MI355X, a copy with non-temporal loads and stores moves about 6.2 TB/s
// against 5.4-5.6 TB/s with ordinary ones.
// ---------------------------------------------------------------------------
__device__ __forceinline__ u32x4_t ld_stream(const u32x4_t* p) {
  return __builtin_nontemporal_load(p);
}
__device__ __forceinline__ void st_stream(u32x4_t* p, const u32x4_t& v) {
  __builtin_nontemporal_store(v, p);
}
__device__ __forceinline__ f32x4_t ld_stream(const f32x4_t* p) {
  return __builtin_nontemporal_load(p);
}
__device__ __forceinline__ void st_stream(f32x4_t* p, const f32x4_t& v) {
  __builtin_nontemporal_store(v, p);
}

// ---------------------------------------------------------------------------
// Element traits: load 8 consecutive values as float, store 8 from float.
// All activation rows are 16-byte aligned and a multiple of 8 elements.
// ---------------------------------------------------------------------------
template <typename T> struct Elem;

template <> struct Elem<float> {
  static constexpr int kBytes = 4;
  __device__ static __forceinline__ void load8(const float* p, float v[8]) {
    f32x4_t a = *reinterpret_cast<const f32x4_t*>(p);
    f32x4_t b = *reinterpret_cast<const f32x4_t*>(p + 4);
    v[0] = a[0]; v[1] = a[1]; v[2] = a[2]; v[3] = a[3];
    v[4] = b[0]; v[5] = b[1]; v[6] = b[2]; v[7] = b[3];
  }
  __device__ static __forceinline__ void store8(float* p, const float v[8]) {
    f32x4_t a = {v[0], v[1], v[2], v[3]};
    f32x4_t b = {v[4], v[5], v[6], v[7]};
    *reinterpret_cast<f32x4_t*>(p) = a;
    *reinterpret_cast<f32x4_t*>(p + 4) = b;
  }
  __device__ static __forceinline__ void load8_stream(const float* p, float v[8]) {
    f32x4_t a = ld_stream(reinterpret_cast<const f32x4_t*>(p));
    f32x4_t b = ld_stream(reinterpret_cast<const f32x4_t*>(p + 4));
    v[0] = a[0]; v[1] = a[1]; v[2] = a[2]; v[3] = a[3];
    v[4] = b[0]; v[5] = b[1]; v[6] = b[2]; v[7] = b[3];
  }
  __device__ static __forceinline__ void store8_stream(float* p, const float v[8]) {
    st_stream(reinterpret_cast<f32x4_t*>(p), f32x4_t{v[0], v[1], v[2], v[3]});
    st_stream(reinterpret_cast<f32x4_t*>(p + 4), f32x4_t{v[4], v[5], v[6], v[7]});
  }
};

template <> struct Elem<bf16_t> {
  static constexpr int kBytes = 2;
  __device__ static __forceinline__ void load8(const bf16_t* p, float v[8]) {
    u32x4_t w = *reinterpret_cast<const u32x4_t*>(p);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      v[2 * i] = lo_bf16(w[i]);
      v[2 * i + 1] = hi_bf16(w[i]);
    }
  }
  __device__ static __forceinline__ void store8(bf16_t* p, const float v[8]) {
    u32x4_t w;
#pragma unroll
    for (int i = 0; i < 4; ++i) w[i] = pack_bf16x2(v[2 * i], v[2 * i + 1]);
    *reinterpret_cast<u32x4_t*>(p) = w;
  }
  __device__ static __forceinline__ void load8_stream(const bf16_t* p, float v[8]) {
    u32x4_t w = ld_stream(reinterpret_cast<const u32x4_t*>(p));
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      v[2 * i] = lo_bf16(w[i]);
      v[2 * i + 1] = hi_bf16(w[i]);
    }
  }
  __device__ static __forceinline__ void store8_stream(bf16_t* p, const float v[8]) {
    u32x4_t w;
#pragma unroll
    for (int i = 0; i < 4; ++i) w[i] = pack_bf16x2(v[2 * i], v[2 * i + 1]);
    st_stream(reinterpret_cast<u32x4_t*>(p), w);
  }
};

// ---------------------------------------------------------------------------
// Wave-level helpers
// ---------------------------------------------------------------------------
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, kWave);
  return v;
}

__device__ __forceinline__ uint64_t lanemask_lt() {
  const int lane = threadIdx.x & (kWave - 1);
  return lane == 0 ? 0ull : (~0ull >> (64 - lane));
}

// sigmoid / SiLU for bf16 outputs: hardware exp2 and reciprocal (about 1 ulp
// each in fp32, far below bf16 resolution)
__device__ __forceinline__ float fast_sigmoid(float a) {
  return __builtin_amdgcn_rcpf(1.0f + __expf(-a));
}
__device__ __forceinline__ float fast_silu(float a) { return a * fast_sigmoid(a); }

}  // namespace laep
