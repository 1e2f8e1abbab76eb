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

// float -> bfloat16, round to nearest even (v_cvt_pk_bf16_f32).
typedef __attribute__((__vector_size__(2 * sizeof(float)))) float f32x2_t;
typedef __attribute__((__vector_size__(2 * sizeof(__bf16)))) __bf16 bf16x2_t;
RAVEL_DEV uint32_t pack_bf16x2(float lo, float hi) {
  const bf16x2_t r = __builtin_convertvector((f32x2_t{lo, hi}), bf16x2_t);
  return __builtin_bit_cast(uint32_t, r);
}
RAVEL_DEV bf16_t f32_to_bf16(float f) { return (bf16_t)(pack_bf16x2(f, 0.f) & 0xFFFFu); }

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

// gelu_tanh(x) = 0.5 x (1 + tanh(u)) with u = sqrt(2/pi) (x + 0.044715 x^3), written
// as x / (1 + exp(-2u)) (the same function: 1 + tanh(u) = 2 / (1 + exp(-2u))) and
// evaluated with the hardware exp2 and reciprocal, a few ulp; large |x| saturate to
// x and to -0.
RAVEL_DEV float gelu_tanh_f(float x) {
  const float c = -2.0f * 0.7978845608028654f * 1.4426950408889634f;  // -2 sqrt(2/pi) log2(e)
  const float t = c * x * (1.0f + 0.044715f * x * x);
  return x * __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(t));
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

// ---------------------------------------------------------------------------
// Cross-block hand-off inside one kernel ("last block reduces").
//
// An agent-scope release/acquire fence on gfx950 writes back and invalidates
// the issuing XCD's whole L2; issued by hundreds of blocks it serialises
// (measured ~0.13 us per block).  Instead, exchanged data is written and read
// with relaxed device-scope atomics, which the compiler emits as device-
// coherent accesses (sc1), every thread waits for its own stores to complete
// before the block takes its ticket, and only the block that takes the last
// ticket reads the other blocks' data.  Nothing ever spins.
// ---------------------------------------------------------------------------
// Pointers in the global address space: atomics on generic pointers become
// flat instructions, which also count against the LDS counter (every later LDS
// wait then waits for them) and cannot be widened.
#define RAVEL_GLOBAL __attribute__((address_space(1)))
template <class T>
RAVEL_DEV RAVEL_GLOBAL T* gptr(T* p) {
  return (RAVEL_GLOBAL T*)p;
}
RAVEL_DEV void coherent_store(float* p, float v) {
  __hip_atomic_store(gptr(p), v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
RAVEL_DEV float coherent_load(const float* p) {
  return __hip_atomic_load(gptr(const_cast<float*>(p)), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
RAVEL_DEV void coherent_store4(float* p, f32x4_t v) {
  uint64_t* q = reinterpret_cast<uint64_t*>(p);
  const u32x4_t u = __builtin_bit_cast(u32x4_t, v);
  __hip_atomic_store(gptr(q), (uint64_t)u[0] | ((uint64_t)u[1] << 32), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  __hip_atomic_store(gptr(q + 1), (uint64_t)u[2] | ((uint64_t)u[3] << 32), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
RAVEL_DEV f32x4_t coherent_load4(const float* p) {
  uint64_t* q = reinterpret_cast<uint64_t*>(const_cast<float*>(p));
  const uint64_t lo = __hip_atomic_load(gptr(q), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  const uint64_t hi = __hip_atomic_load(gptr(q + 1), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  const u32x4_t u = {(uint32_t)lo, (uint32_t)(lo >> 32), (uint32_t)hi, (uint32_t)(hi >> 32)};
  return __builtin_bit_cast(f32x4_t, u);
}
// Wait until this thread's outstanding memory operations have completed.
RAVEL_DEV void wait_memory() {
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
  __builtin_amdgcn_s_waitcnt(0);
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
}
// After winning the last ticket: drop this CU's and XCD's cached copies so that
// plain (pipelined) loads fetch the other blocks' write-through data.  An
// agent-scope acquire fence only invalidates (no L2 write-back).
RAVEL_DEV void acquire_device() { __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "agent"); }
// All threads of the block call this after their coherent stores; returns true
// (uniformly) in the block that arrives last of `arrivals`, which also re-arms
// the counter for the next launch.
RAVEL_DEV bool last_block_arrival(unsigned* counter, unsigned arrivals, int* s_flag) {
  wait_memory();
  __syncthreads();
  if (threadIdx.x == 0) {
    const unsigned prev = __hip_atomic_fetch_add(gptr(counter), 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    *s_flag = (prev == arrivals - 1);
    if (prev == arrivals - 1)
      __hip_atomic_store(gptr(counter), 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
  __syncthreads();
  const bool last = *s_flag != 0;
  if (last) acquire_device();
  return last;
}
