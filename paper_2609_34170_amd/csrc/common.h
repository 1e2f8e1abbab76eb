// Shared device helpers for the CDNA4 (gfx950) kernels of libravel.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

typedef uint16_t bf16_t;  // raw bfloat16 bits

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8_t;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4_t;
typedef __attribute__((__vector_size__(4 * sizeof(uint32_t)))) uint32_t u32x4_t;
typedef __attribute__((__vector_size__(2 * sizeof(uint32_t)))) uint32_t u32x2_t;

#define RAVEL_DEV __device__ __forceinline__

RAVEL_DEV float bf16_to_f32(bf16_t h) { return __uint_as_float(((uint32_t)h) << 16); }

// float -> bfloat16, round to nearest even (inputs here are finite).
RAVEL_DEV bf16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (bf16_t)(u >> 16);
}

// Activation element type traits: float (fp32 models) or bf16_t.
template <typename T> struct act;
template <> struct act<float> {
  static RAVEL_DEV float load(const float* p) { return *p; }
  static RAVEL_DEV float to_f(float v) { return v; }
  static RAVEL_DEV float from_f(float v) { return v; }
};
template <> struct act<bf16_t> {
  static RAVEL_DEV float load(const bf16_t* p) { return bf16_to_f32(*p); }
  static RAVEL_DEV float to_f(bf16_t v) { return bf16_to_f32(v); }
  static RAVEL_DEV bf16_t from_f(float v) { return f32_to_bf16(v); }
};

RAVEL_DEV float silu_f(float x) { return x / (1.0f + __expf(-x)); }

RAVEL_DEV float gelu_tanh_f(float x) {
  const float c = 0.7978845608028654f;  // sqrt(2/pi)
  float u = c * (x + 0.044715f * x * x * x);
  return 0.5f * x * (1.0f + tanhf(u));
}

// Sum across the 64 lanes of a wavefront.
RAVEL_DEV float wave_sum(float v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}
RAVEL_DEV float wave_max(float v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v = fmaxf(v, __shfl_xor(v, off, 64));
  return v;
}
