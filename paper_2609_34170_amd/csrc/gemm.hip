// GEMM kernels: C[M,N] = A[M,K] . B[N,K]^T with fused epilogues.
//
// bf16 path: LDS-tiled MFMA kernel (v_mfma_f32_16x16x32_bf16, wave64, 4 waves
// per block), double-buffered LDS with register prefetch of the next K tile,
// and an optional deterministic split-K: every K range writes its fp32
// partial tile, the last block to arrive (device-scope ticket) sums the
// partials in fixed range order and runs the epilogue.
//
// fp32 path: a plain SIMT kernel (one output per thread) for the small fp32
// models, which are latency bound.
#include "kernels.h"

namespace ravel {

template <typename T>
RAVEL_DEV void epi_store(const GemmArgs& a, int m, int n, float acc) {
  const float b = a.bias ? a.bias[n] : 0.0f;
  switch (a.mode) {
    case EPI_F32:
      a.out_f[(size_t)m * a.ldo_f + n] = acc + b;
      break;
    case EPI_T:
      ((T*)a.out_t)[(size_t)m * a.ldo_t + n] = act<T>::from_f(acc + b);
      break;
    case EPI_RESID: {
      const float g = a.gate ? a.gate[(size_t)m * a.ldg + n] : 1.0f;
      float* o = a.out_f + (size_t)m * a.ldo_f + n;
      *o = *o + g * acc;
      break;
    }
    case EPI_RESID_TANH: {
      const float g = tanhf(*a.gate_scalar);
      float* o = a.out_f + (size_t)m * a.ldo_f + n;
      *o = *o + g * acc;
      break;
    }
    case EPI_COND: {
      const float base = acc + b;
      for (int i = 0; i < a.H; ++i)
        ((T*)a.out_t)[((size_t)m * a.H + i) * a.ldo_t + n] =
            act<T>::from_f(silu_f(a.ctau[(size_t)i * a.N + n] + base));
      break;
    }
    case EPI_GELU_T:
      ((T*)a.out_t)[(size_t)m * a.ldo_t + n] = act<T>::from_f(gelu_tanh_f(acc + b));
      break;
    case EPI_SILU_T:
      ((T*)a.out_t)[(size_t)m * a.ldo_t + n] = act<T>::from_f(silu_f(acc + b));
      break;
    default:
      break;
  }
}

template <typename T>
RAVEL_DEV void epi_geglu(const GemmArgs& a, int m, int f, float g, float u) {
  ((T*)a.out_t)[(size_t)m * a.ldo_t + f] = act<T>::from_f(gelu_tanh_f(g) * u);
}

// ---------------------------------------------------------------------------
// bf16 MFMA kernel
// ---------------------------------------------------------------------------
template <int BM, int BN, int WM, int WN>
__global__ __launch_bounds__(256) void gemm_bf16_kernel(GemmArgs a) {
  constexpr int BK = 64;
  constexpr int LDK = BK + 8;  // +16 bytes per row: conflict-free 16-byte fragment reads
  constexpr int TM = BM / (16 * WM);
  constexpr int TN = BN / (16 * WN);
  constexpr int CA = BM * (BK / 8) / 256;  // 16-byte chunks per thread, A tile
  constexpr int CB = BN * (BK / 8) / 256;
  static_assert(WM * WN == 4, "4 waves");
  static_assert(CA >= 1 && CB >= 1, "tile too small");

  __shared__ __attribute__((aligned(16))) bf16_t As[2][BM][LDK];
  __shared__ __attribute__((aligned(16))) bf16_t Bs[2][BN][LDK];
  __shared__ int s_last;

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int l16 = lane & 15, grp = lane >> 4;
  const int wm = wave / WN, wn = wave % WN;

  const int tiles_n = (a.N + BN - 1) / BN;
  const int tile = blockIdx.x;
  const int m0 = (tile / tiles_n) * BM;
  const int n0 = (tile % tiles_n) * BN;
  const int z = blockIdx.z;
  const int kbeg = z * a.kchunk;
  const int kend = min(a.K, kbeg + a.kchunk);
  const int nk = (kend - kbeg + BK - 1) / BK;

  const bf16_t* __restrict__ A = (const bf16_t*)a.A;
  const bf16_t* __restrict__ B = (const bf16_t*)a.B;

  u32x4_t ra[CA], rb[CB];
  auto gload = [&](int kt) {
    const int k0 = kbeg + kt * BK;
#pragma unroll
    for (int i = 0; i < CA; ++i) {
      const int c = tid + i * 256;
      const int row = c >> 3, kc = (c & 7) * 8;
      const int m = m0 + row, k = k0 + kc;
      if (m < a.M && k < kend)
        ra[i] = *(const u32x4_t*)(A + (size_t)m * a.lda + k);
      else
        ra[i] = u32x4_t{0, 0, 0, 0};
    }
#pragma unroll
    for (int i = 0; i < CB; ++i) {
      const int c = tid + i * 256;
      const int row = c >> 3, kc = (c & 7) * 8;
      const int n = n0 + row, k = k0 + kc;
      if (n < a.N && k < kend)
        rb[i] = *(const u32x4_t*)(B + (size_t)n * a.ldb + k);
      else
        rb[i] = u32x4_t{0, 0, 0, 0};
    }
  };
  auto sstore = [&](int buf) {
#pragma unroll
    for (int i = 0; i < CA; ++i) {
      const int c = tid + i * 256;
      *(u32x4_t*)&As[buf][c >> 3][(c & 7) * 8] = ra[i];
    }
#pragma unroll
    for (int i = 0; i < CB; ++i) {
      const int c = tid + i * 256;
      *(u32x4_t*)&Bs[buf][c >> 3][(c & 7) * 8] = rb[i];
    }
  };

  f32x4_t acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  if (nk > 0) {
    gload(0);
    sstore(0);
  }
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < nk) gload(kt + 1);
#pragma unroll
    for (int ks = 0; ks < BK / 32; ++ks) {
      bf16x8_t af[TM], bfr[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i)
        af[i] = *(const bf16x8_t*)&As[buf][wm * (BM / WM) + i * 16 + l16][ks * 32 + grp * 8];
#pragma unroll
      for (int j = 0; j < TN; ++j)
        bfr[j] = *(const bf16x8_t*)&Bs[buf][wn * (BN / WN) + j * 16 + l16][ks * 32 + grp * 8];
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
    }
    if (kt + 1 < nk) sstore(buf ^ 1);
    __syncthreads();
  }

  // acc[i][j][r] = C[m0 + wm*(BM/WM) + i*16 + grp*4 + r][n0 + wn*(BN/WN) + j*16 + l16]
  const int mw = m0 + wm * (BM / WM);
  const int nw = n0 + wn * (BN / WN);

  if (a.ksplit > 1) {
    float* part = a.partial + (size_t)z * a.M * a.N;
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int m = mw + i * 16 + grp * 4 + r, n = nw + j * 16 + l16;
          if (m < a.M && n < a.N) part[(size_t)m * a.N + n] = acc[i][j][r];
        }
    __threadfence();
    __syncthreads();
    if (tid == 0) {
      unsigned prev = __hip_atomic_fetch_add(&a.counters[tile * kCounterStride], 1u, __ATOMIC_ACQ_REL,
                                             __HIP_MEMORY_SCOPE_AGENT);
      s_last = (prev == (unsigned)(a.ksplit - 1));
    }
    __syncthreads();
    if (!s_last) return;
    __threadfence();
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int m = mw + i * 16 + grp * 4 + r, n = nw + j * 16 + l16;
          if (m < a.M && n < a.N) {
            float s = 0.f;
            for (int zz = 0; zz < a.ksplit; ++zz)
              s += (zz == z) ? acc[i][j][r]
                             : a.partial[((size_t)zz * a.M + m) * a.N + n];
            acc[i][j][r] = s;
          }
        }
    if (tid == 0) a.counters[tile * kCounterStride] = 0u;
  }

  if constexpr (TN % 2 == 0) {
    if (a.mode == EPI_GEGLU) {
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; j += 2)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int m = mw + i * 16 + grp * 4 + r;
          const int ng = nw + j * 16;  // gate block start, multiple of 32
          const int f = (ng >> 5) * 16 + l16;
          if (m < a.M && ng < a.N)
            epi_geglu<bf16_t>(a, m, f, acc[i][j][r], acc[i][j + 1][r]);
        }
      return;
    }
  }
  {
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int m = mw + i * 16 + grp * 4 + r, n = nw + j * 16 + l16;
          if (m < a.M && n < a.N) epi_store<bf16_t>(a, m, n, acc[i][j][r]);
        }
  }
}

template <int BM, int BN, int WM, int WN>
static hipError_t launch_tile(const GemmArgs& a, hipStream_t s) {
  const int tiles = ((a.M + BM - 1) / BM) * ((a.N + BN - 1) / BN);
  dim3 grid(tiles, 1, a.ksplit);
  hipLaunchKernelGGL((gemm_bf16_kernel<BM, BN, WM, WN>), grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_gemm_bf16(const GemmArgs& a, int tile, hipStream_t s) {
  switch (tile) {
    case TILE_128x128: return launch_tile<128, 128, 2, 2>(a, s);
    case TILE_64x128: return launch_tile<64, 128, 2, 2>(a, s);
    case TILE_128x64: return launch_tile<128, 64, 2, 2>(a, s);
    case TILE_32x64: return launch_tile<32, 64, 1, 4>(a, s);
    case TILE_64x64:
    default: return launch_tile<64, 64, 2, 2>(a, s);
  }
}

// ---------------------------------------------------------------------------
// fp32 SIMT kernel
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void gemm_f32_kernel(GemmArgs a) {
  const int n = blockIdx.x * 64 + (threadIdx.x & 63);
  const int m = blockIdx.y * 4 + (threadIdx.x >> 6);
  if (m >= a.M) return;
  const float* __restrict__ A = (const float*)a.A + (size_t)m * a.lda;
  const float* __restrict__ B = (const float*)a.B;
  if (a.mode == EPI_GEGLU) {
    const int F = a.N / 2;
    if (n >= F) return;
    const int rg = (n >> 4) * 32 + (n & 15);
    const float* bg = B + (size_t)rg * a.ldb;
    const float* bu = B + (size_t)(rg + 16) * a.ldb;
    float g = 0.f, u = 0.f;
    for (int k = 0; k < a.K; ++k) {
      g += A[k] * bg[k];
      u += A[k] * bu[k];
    }
    epi_geglu<float>(a, m, n, g, u);
  } else {
    if (n >= a.N) return;
    const float* b = B + (size_t)n * a.ldb;
    float acc = 0.f;
    for (int k = 0; k < a.K; ++k) acc += A[k] * b[k];
    epi_store<float>(a, m, n, acc);
  }
}

hipError_t launch_gemm_f32(const GemmArgs& a, hipStream_t s) {
  const int ncols = a.mode == EPI_GEGLU ? a.N / 2 : a.N;
  dim3 grid((ncols + 63) / 64, (a.M + 3) / 4);
  hipLaunchKernelGGL(gemm_f32_kernel, grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace ravel
