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
#include <algorithm>

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
    // split-K: fragment-native partials (each lane writes/reads 16 contiguous bytes)
    const size_t tile_elems = (size_t)BM * BN;
    float* part = a.partial + ((size_t)z * gridDim.x + tile) * tile_elems;
    const int wbase = (wave * TM * TN) * 256;
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j) coherent_store4(part + wbase + ((i * TN + j) * 64 + lane) * 4, acc[i][j]);
    if (!last_block_arrival(&a.counters[tile * kCounterStride], (unsigned)a.ksplit, &s_last)) return;
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        f32x4_t sum = {0.f, 0.f, 0.f, 0.f};
        for (int zz = 0; zz < a.ksplit; ++zz) {
          const f32x4_t v = (zz == z) ? acc[i][j]
                                      : *(const f32x4_t*)(a.partial + ((size_t)zz * gridDim.x + tile) * tile_elems + wbase +
                                                          ((i * TN + j) * 64 + lane) * 4);
          sum[0] += v[0];
          sum[1] += v[1];
          sum[2] += v[2];
          sum[3] += v[3];
        }
        acc[i][j] = sum;
      }
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


// ---------------------------------------------------------------------------
// Weight-streaming kernel for few rows (M <= 64): the regime of one env's H
// slots, where every weight byte is used by at most 64 rows and the GEMM is
// bound by streaming the weights from HBM.
//
// Block = 4 waves, block tile = (4 x NFR x 16) output columns x all M rows x
// one K range of KR (grid.y).  The MFMA runs with the weights as its A
// operand (C^T = W A^T) so that each lane owns 4 consecutive output columns
// of one row and the epilogue writes 16-byte vectors.  Each wave issues all
// weight fragments of a tile at once; the activations of the K range are
// staged in LDS once per block, and blocks loop over column tiles
// (grid.x may be smaller than the tile count), issuing the next tile's weight
// loads before the current tile's epilogue.  Split-K ranges are reduced by the
// last-arriving block of a tile, in fixed order.
// ---------------------------------------------------------------------------
template <typename T>
RAVEL_DEV void epi_store4(const GemmArgs& a, int m, int n, f32x4_t acc) {
  // n .. n+3 are valid columns of row m (N is a multiple of 4)
  f32x4_t b = {0.f, 0.f, 0.f, 0.f};
  if (a.bias) b = *(const f32x4_t*)(a.bias + n);
  switch (a.mode) {
    case EPI_F32: {
      f32x4_t o = {acc[0] + b[0], acc[1] + b[1], acc[2] + b[2], acc[3] + b[3]};
      *(f32x4_t*)(a.out_f + (size_t)m * a.ldo_f + n) = o;
      break;
    }
    case EPI_RESID:
    case EPI_RESID_TANH: {
      f32x4_t g = {1.f, 1.f, 1.f, 1.f};
      if (a.mode == EPI_RESID_TANH) {
        const float t = tanhf(*a.gate_scalar);
        g = f32x4_t{t, t, t, t};
      } else if (a.gate) {
        g = *(const f32x4_t*)(a.gate + (size_t)m * a.ldg + n);
      }
      f32x4_t* o = (f32x4_t*)(a.out_f + (size_t)m * a.ldo_f + n);
      f32x4_t x = *o;
      x[0] = x[0] + g[0] * acc[0];
      x[1] = x[1] + g[1] * acc[1];
      x[2] = x[2] + g[2] * acc[2];
      x[3] = x[3] + g[3] * acc[3];
      *o = x;
      break;
    }
    case EPI_T: {
      if constexpr (sizeof(T) == 2) {
        u32x2_t w;
        w[0] = (uint32_t)f32_to_bf16(acc[0] + b[0]) | ((uint32_t)f32_to_bf16(acc[1] + b[1]) << 16);
        w[1] = (uint32_t)f32_to_bf16(acc[2] + b[2]) | ((uint32_t)f32_to_bf16(acc[3] + b[3]) << 16);
        *(u32x2_t*)((bf16_t*)a.out_t + (size_t)m * a.ldo_t + n) = w;
        break;
      }
    }
      [[fallthrough]];
    default:
#pragma unroll
      for (int r = 0; r < 4; ++r) epi_store<T>(a, m, n + r, acc[r]);
      break;
  }
}

// Whether the 4-column vector epilogue applies to this launch (alignment of every
// row stride it touches).
RAVEL_DEV bool epi_vec_ok(const GemmArgs& a) {
  switch (a.mode) {
    case EPI_F32: return (a.ldo_f % 4) == 0;
    case EPI_RESID: return (a.ldo_f % 4) == 0 && (!a.gate || (a.ldg % 4) == 0);
    case EPI_RESID_TANH: return (a.ldo_f % 4) == 0;
    case EPI_T: return (a.ldo_t % 4) == 0;
    default: return true;
  }
}

template <int MT, int NFR, int KR>
__global__ __launch_bounds__(256) void gemm_skinny_kernel(GemmArgs a) {
  constexpr int NF = KR / 32;  // weight fragments per lane per 16-column block
  constexpr int LDA = KR + 8;
  __shared__ __attribute__((aligned(16))) bf16_t As[MT * 16][LDA];
  __shared__ int s_last;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l16 = lane & 15, grp = lane >> 4;
  const int z = blockIdx.y;
  const int kbeg = z * KR;
  const int tiles = (a.N + 64 * NFR - 1) / (64 * NFR);
  const bf16_t* __restrict__ A = (const bf16_t*)a.A;
  const bf16_t* __restrict__ B = (const bf16_t*)a.B;

  bf16x8_t wfr[NFR][NF];
  auto load_w = [&](int tile) {
    const int nw = tile * (64 * NFR) + wave * (16 * NFR);
#pragma unroll
    for (int c = 0; c < NFR; ++c) {
      const int n = nw + c * 16 + l16;
#pragma unroll
      for (int f = 0; f < NF; ++f) {
        const int k = kbeg + f * 32 + grp * 8;
        if (n < a.N && k < a.K)
          wfr[c][f] = *(const bf16x8_t*)(B + (size_t)n * a.ldb + k);
        else
          wfr[c][f] = bf16x8_t{};
      }
    }
  };
  int tile = blockIdx.x;
  if (tile >= tiles) return;
  load_w(tile);

  // activations of the K range -> LDS, loads issued in batches of 8 per thread
  constexpr int CA = (MT * 16 * (KR / 8) + 255) / 256;
  constexpr int BATCH = CA < 8 ? CA : 8;
#pragma unroll
  for (int b0 = 0; b0 < CA; b0 += BATCH) {
    u32x4_t av[BATCH];
#pragma unroll
    for (int i = 0; i < BATCH; ++i) {
      const int c = tid + (b0 + i) * 256;
      const int row = c / (KR / 8), kc = (c % (KR / 8)) * 8;
      const int k = kbeg + kc;
      av[i] = u32x4_t{0, 0, 0, 0};
      if (c < MT * 16 * (KR / 8) && row < a.M && k < a.K) av[i] = *(const u32x4_t*)(A + (size_t)row * a.lda + k);
    }
#pragma unroll
    for (int i = 0; i < BATCH; ++i) {
      const int c = tid + (b0 + i) * 256;
      if (c < MT * 16 * (KR / 8)) *(u32x4_t*)&As[c / (KR / 8)][(c % (KR / 8)) * 8] = av[i];
    }
  }
  __syncthreads();

  for (; tile < tiles; tile += gridDim.x) {
    const int nw = tile * (64 * NFR) + wave * (16 * NFR);
    f32x4_t acc[NFR][MT];
#pragma unroll
    for (int c = 0; c < NFR; ++c)
#pragma unroll
      for (int i = 0; i < MT; ++i) acc[c][i] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int f = 0; f < NF; ++f) {
#pragma unroll
      for (int i = 0; i < MT; ++i) {
        const bf16x8_t xf = *(const bf16x8_t*)&As[i * 16 + l16][f * 32 + grp * 8];
#pragma unroll
        for (int c = 0; c < NFR; ++c)
          acc[c][i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wfr[c][f], xf, acc[c][i], 0, 0, 0);
      }
    }
    // overlap: the next tile's weights stream in during this tile's epilogue
    if (tile + (int)gridDim.x < tiles) load_w(tile + gridDim.x);

    if (a.ksplit > 1) {
      constexpr int FR = MT * NFR;  // fragments per wave
      const size_t tile_elems = (size_t)4 * FR * 256;
      const int wbase = wave * FR * 256;
      float* part = a.partial + ((size_t)z * tiles + tile) * tile_elems;
#pragma unroll
      for (int c = 0; c < NFR; ++c)
#pragma unroll
        for (int i = 0; i < MT; ++i) coherent_store4(part + wbase + ((c * MT + i) * 64 + lane) * 4, acc[c][i]);
      if (!last_block_arrival(&a.counters[tile * kCounterStride], (unsigned)a.ksplit, &s_last)) continue;
#pragma unroll
      for (int c = 0; c < NFR; ++c)
#pragma unroll
        for (int i = 0; i < MT; ++i) {
          f32x4_t sum = {0.f, 0.f, 0.f, 0.f};
          for (int zz = 0; zz < a.ksplit; ++zz) {
            const f32x4_t v = (zz == z) ? acc[c][i]
                                        : *(const f32x4_t*)(a.partial + ((size_t)zz * tiles + tile) * tile_elems +
                                                            wbase + ((c * MT + i) * 64 + lane) * 4);
            sum[0] += v[0];
            sum[1] += v[1];
            sum[2] += v[2];
            sum[3] += v[3];
          }
          acc[c][i] = sum;
        }
    }

    // acc[c][i][r] = C[m = i*16 + l16][n = nw + c*16 + 4*grp + r]
    bool done = false;
    if constexpr (NFR % 2 == 0) {
      if (a.mode == EPI_GEGLU) {
#pragma unroll
        for (int c = 0; c < NFR; c += 2)
#pragma unroll
          for (int i = 0; i < MT; ++i) {
            const int m = i * 16 + l16;
            const int ng = nw + c * 16;  // gate block start (multiple of 32)
            if (m < a.M && ng < a.N) {
              const int f = (ng >> 5) * 16 + grp * 4;
              u32x2_t w;
              w[0] = (uint32_t)f32_to_bf16(gelu_tanh_f(acc[c][i][0]) * acc[c + 1][i][0]) |
                     ((uint32_t)f32_to_bf16(gelu_tanh_f(acc[c][i][1]) * acc[c + 1][i][1]) << 16);
              w[1] = (uint32_t)f32_to_bf16(gelu_tanh_f(acc[c][i][2]) * acc[c + 1][i][2]) |
                     ((uint32_t)f32_to_bf16(gelu_tanh_f(acc[c][i][3]) * acc[c + 1][i][3]) << 16);
              *(u32x2_t*)((bf16_t*)a.out_t + (size_t)m * a.ldo_t + f) = w;
            }
          }
        done = true;
      }
    }
    if (!done) {
      const bool vec = epi_vec_ok(a);
#pragma unroll
      for (int c = 0; c < NFR; ++c)
#pragma unroll
        for (int i = 0; i < MT; ++i) {
          const int m = i * 16 + l16, n = nw + c * 16 + grp * 4;
          if (m >= a.M || n >= a.N) continue;
          if (vec && n + 4 <= a.N) {
            epi_store4<bf16_t>(a, m, n, acc[c][i]);
          } else {
#pragma unroll
            for (int r = 0; r < 4; ++r)
              if (n + r < a.N) epi_store<bf16_t>(a, m, n + r, acc[c][i][r]);
          }
        }
    }
  }
}

template <int MT, int NFR, int KR>
static hipError_t launch_skinny_t(const GemmArgs& a, hipStream_t s) {
  const int tiles = (a.N + 64 * NFR - 1) / (64 * NFR);
  // at most ~2 resident waves of blocks; extra tiles are looped over inside a block
  const int cap = (a.ksplit > 1) ? tiles : std::max(1, std::min(tiles, 512));
  dim3 grid(cap, a.ksplit);
  hipLaunchKernelGGL((gemm_skinny_kernel<MT, NFR, KR>), grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

template <int MT>
static hipError_t launch_skinny_m(const GemmArgs& a, int nfr, hipStream_t s) {
  switch (a.kchunk) {
    case 128: return nfr == 2 ? launch_skinny_t<MT, 2, 128>(a, s) : launch_skinny_t<MT, 1, 128>(a, s);
    case 256: return nfr == 2 ? launch_skinny_t<MT, 2, 256>(a, s) : launch_skinny_t<MT, 1, 256>(a, s);
    case 512: return nfr == 2 ? launch_skinny_t<MT, 2, 512>(a, s) : launch_skinny_t<MT, 1, 512>(a, s);
    case 1024: return nfr == 1 ? launch_skinny_t<MT, 1, 1024>(a, s) : hipErrorInvalidValue;
    default: return hipErrorInvalidValue;
  }
}

hipError_t launch_gemm_skinny(const GemmArgs& a, int nfr, hipStream_t s) {
  if (a.M > 64 || (a.mode == EPI_GEGLU && (nfr != 2 || a.N % 32))) return hipErrorInvalidValue;
  if (a.ksplit * a.kchunk < a.K) return hipErrorInvalidValue;
  switch ((a.M + 15) / 16) {
    case 1: return launch_skinny_m<1>(a, nfr, s);
    case 2: return launch_skinny_m<2>(a, nfr, s);
    case 3: return launch_skinny_m<3>(a, nfr, s);
    default: return launch_skinny_m<4>(a, nfr, s);
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
