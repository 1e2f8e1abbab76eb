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

// Epilogues.  Every MFMA result fragment here holds 4 consecutive output columns
// n .. n+3 of one row m per lane; epilogues are specialised by mode so that the
// fully unrolled fragment loops stay small (a large inlined switch there makes
// the compiler keep the accumulators in scratch memory).
template <int MODE, typename T>
RAVEL_DEV void epi1(const GemmArgs& a, int m, int n, float acc) {
  const float b = a.bias ? a.bias[n] : 0.0f;
  if constexpr (MODE == EPI_F32) {
    a.out_f[(size_t)m * a.ldo_f + n] = acc + b;
  } else if constexpr (MODE == EPI_T) {
    ((T*)a.out_t)[(size_t)m * a.ldo_t + n] = act<T>::from_f(acc + b);
  } else if constexpr (MODE == EPI_RESID) {
    const size_t gm = a.gate_rows ? (size_t)a.gate_rows[m] : (size_t)m;
    const float g = a.gate ? a.gate[gm * a.ldg + n] : 1.0f;
    float* o = a.out_f + (size_t)m * a.ldo_f + n;
    *o = *o + g * acc;
  } else if constexpr (MODE == EPI_RESID_TANH) {
    float* o = a.out_f + (size_t)m * a.ldo_f + n;
    *o = *o + tanhf(*a.gate_scalar) * acc;
  } else if constexpr (MODE == EPI_COND) {
    const int blk = a.cond_grp ? a.cond_grp[m] : m;
    if (blk < 0) return;
    const float base = acc + b;
    for (int i = 0; i < a.H; ++i)
      ((T*)a.out_t)[((size_t)blk * a.H + i) * a.ldo_t + n] = act<T>::from_f(silu_f(a.ctau[(size_t)i * a.N + n] + base));
  } else if constexpr (MODE == EPI_GELU_T) {
    ((T*)a.out_t)[(size_t)m * a.ldo_t + n] = act<T>::from_f(gelu_tanh_f(acc + b));
  } else if constexpr (MODE == EPI_SILU_T) {
    ((T*)a.out_t)[(size_t)m * a.ldo_t + n] = act<T>::from_f(silu_f(acc + b));
  }
}

// Whether the 4-column vector path applies to this launch (row strides aligned).
RAVEL_DEV bool epi_vec_ok(const GemmArgs& a) {
  switch (a.mode) {
    case EPI_F32: return (a.ldo_f % 4) == 0;
    case EPI_RESID: return (a.ldo_f % 4) == 0 && (!a.gate || (a.ldg % 4) == 0);
    case EPI_RESID_TANH: return (a.ldo_f % 4) == 0;
    case EPI_T:
    case EPI_GELU_T:
    case EPI_SILU_T: return (a.ldo_t % 4) == 0;
    case EPI_COND: return (a.ldo_t % 4) == 0 && (a.N % 4) == 0;
    default: return true;
  }
}

RAVEL_DEV void store_bf16x4(bf16_t* p, float v0, float v1, float v2, float v3) {
  u32x2_t w;
  w[0] = (uint32_t)f32_to_bf16(v0) | ((uint32_t)f32_to_bf16(v1) << 16);
  w[1] = (uint32_t)f32_to_bf16(v2) | ((uint32_t)f32_to_bf16(v3) << 16);
  *(u32x2_t*)p = w;
}

// bf16 activations; fp32 outputs are written as float4.
template <int MODE>
RAVEL_DEV void epi4(const GemmArgs& a, int m, int n, f32x4_t v, bool vec) {
  if (!(vec && n + 4 <= a.N)) {
#pragma unroll
    for (int r = 0; r < 4; ++r)
      if (n + r < a.N) epi1<MODE, bf16_t>(a, m, n + r, v[r]);
    return;
  }
  f32x4_t b = {0.f, 0.f, 0.f, 0.f};
  if (a.bias) b = *(const f32x4_t*)(a.bias + n);
  if constexpr (MODE == EPI_F32) {
    *(f32x4_t*)(a.out_f + (size_t)m * a.ldo_f + n) = f32x4_t{v[0] + b[0], v[1] + b[1], v[2] + b[2], v[3] + b[3]};
  } else if constexpr (MODE == EPI_T) {
    store_bf16x4((bf16_t*)a.out_t + (size_t)m * a.ldo_t + n, v[0] + b[0], v[1] + b[1], v[2] + b[2], v[3] + b[3]);
  } else if constexpr (MODE == EPI_RESID || MODE == EPI_RESID_TANH) {
    f32x4_t g = {1.f, 1.f, 1.f, 1.f};
    if constexpr (MODE == EPI_RESID_TANH) {
      const float t = tanhf(*a.gate_scalar);
      g = f32x4_t{t, t, t, t};
    } else {
      if (a.gate) g = *(const f32x4_t*)(a.gate + (a.gate_rows ? (size_t)a.gate_rows[m] : (size_t)m) * a.ldg + n);
    }
    f32x4_t* o = (f32x4_t*)(a.out_f + (size_t)m * a.ldo_f + n);
    f32x4_t x = *o;
    x[0] = x[0] + g[0] * v[0];
    x[1] = x[1] + g[1] * v[1];
    x[2] = x[2] + g[2] * v[2];
    x[3] = x[3] + g[3] * v[3];
    *o = x;
  } else if constexpr (MODE == EPI_COND) {
    const int blk = a.cond_grp ? a.cond_grp[m] : m;
    if (blk < 0) return;
    // the time embeddings of 8 slots are loaded before any of their outputs is
    // stored: one memory latency per 8 slots (the stores could alias the loads,
    // so the compiler would otherwise wait for each load in turn)
    for (int i0 = 0; i0 < a.H; i0 += 8) {
      f32x4_t c[8];
#pragma unroll
      for (int j = 0; j < 8; ++j)
        c[j] = (i0 + j < a.H) ? *(const f32x4_t*)(a.ctau + (size_t)(i0 + j) * a.N + n) : f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int j = 0; j < 8; ++j)
        if (i0 + j < a.H)
          store_bf16x4((bf16_t*)a.out_t + ((size_t)blk * a.H + i0 + j) * a.ldo_t + n, silu_f(c[j][0] + v[0] + b[0]),
                       silu_f(c[j][1] + v[1] + b[1]), silu_f(c[j][2] + v[2] + b[2]), silu_f(c[j][3] + v[3] + b[3]));
    }
  } else if constexpr (MODE == EPI_GELU_T) {
    store_bf16x4((bf16_t*)a.out_t + (size_t)m * a.ldo_t + n, gelu_tanh_f(v[0] + b[0]), gelu_tanh_f(v[1] + b[1]),
                 gelu_tanh_f(v[2] + b[2]), gelu_tanh_f(v[3] + b[3]));
  } else if constexpr (MODE == EPI_SILU_T) {
    store_bf16x4((bf16_t*)a.out_t + (size_t)m * a.ldo_t + n, silu_f(v[0] + b[0]), silu_f(v[1] + b[1]),
                 silu_f(v[2] + b[2]), silu_f(v[3] + b[3]));
  }
}

// Gated GeLU of a gate fragment g and its up fragment u: columns f .. f+3 of row m.
RAVEL_DEV void epi_geglu4(const GemmArgs& a, int m, int f, f32x4_t g, f32x4_t u) {
  store_bf16x4((bf16_t*)a.out_t + (size_t)m * a.ldo_t + f, gelu_tanh_f(g[0]) * u[0], gelu_tanh_f(g[1]) * u[1],
               gelu_tanh_f(g[2]) * u[2], gelu_tanh_f(g[3]) * u[3]);
}

// Apply the epilogue to an NI x NJ grid of fragments: fragment (i, j) holds
// rows m0 + 16 i + l16 and columns n0 + 16 j + 4 grp .. +3.
template <int MODE, int NI, int NJ>
RAVEL_DEV void epi_frags(const GemmArgs& a, const f32x4_t (&acc)[NI][NJ], int m0, int n0, int l16, int grp) {
  const bool vec = epi_vec_ok(a);
  if constexpr (MODE == EPI_GEGLU) {
    if constexpr (NJ % 2 == 0) {
#pragma unroll
      for (int i = 0; i < NI; ++i)
#pragma unroll
        for (int j = 0; j < NJ; j += 2) {
          const int m = m0 + i * 16 + l16;
          const int ng = n0 + j * 16;  // gate block start (multiple of 32)
          if (m < a.M && ng < a.N) epi_geglu4(a, m, (ng >> 5) * 16 + grp * 4, acc[i][j], acc[i][j + 1]);
        }
    }
  } else {
#pragma unroll
    for (int i = 0; i < NI; ++i)
#pragma unroll
      for (int j = 0; j < NJ; ++j) {
        const int m = m0 + i * 16 + l16, n = n0 + j * 16 + grp * 4;
        if (m < a.M && n < a.N) epi4<MODE>(a, m, n, acc[i][j], vec);
      }
  }
}

template <int NI, int NJ>
RAVEL_DEV void epilogue(const GemmArgs& a, const f32x4_t (&acc)[NI][NJ], int m0, int n0, int l16, int grp) {
  switch (a.mode) {
    case EPI_F32: epi_frags<EPI_F32>(a, acc, m0, n0, l16, grp); break;
    case EPI_T: epi_frags<EPI_T>(a, acc, m0, n0, l16, grp); break;
    case EPI_RESID: epi_frags<EPI_RESID>(a, acc, m0, n0, l16, grp); break;
    case EPI_RESID_TANH: epi_frags<EPI_RESID_TANH>(a, acc, m0, n0, l16, grp); break;
    case EPI_GEGLU: epi_frags<EPI_GEGLU>(a, acc, m0, n0, l16, grp); break;
    case EPI_COND: epi_frags<EPI_COND>(a, acc, m0, n0, l16, grp); break;
    case EPI_GELU_T: epi_frags<EPI_GELU_T>(a, acc, m0, n0, l16, grp); break;
    case EPI_SILU_T: epi_frags<EPI_SILU_T>(a, acc, m0, n0, l16, grp); break;
    default: break;
  }
}

// ---------------------------------------------------------------------------
// bf16 MFMA kernel
// ---------------------------------------------------------------------------
// Blocks are dispatched round-robin over the 8 XCDs (block b runs on XCD b % 8),
// each with its own L2.  Give every XCD a contiguous range of row-major tiles so
// that the tiles sharing an activation row panel share one L2.
RAVEL_DEV int xcd_tile(int b, int T) {
  const int x = b & 7, local = b >> 3;
  const int q = T >> 3, r = T & 7;  // XCD x owns q + (x < r) tiles
  const int start = x * q + (x < r ? x : r);
  return start + local;
}
// Row and column of tile t of a tiles_m x tiles_n grid ordered in groups of up to 8
// column tiles, row-major inside a group: an XCD's contiguous range of t covers a
// compact rectangle (about 8 x 8 tiles), so its L2 holds the activation row panels and
// the weight column panels it reads instead of every column panel of a wide output.
RAVEL_DEV void tile_rc(int t, int tiles_m, int tiles_n, int& r, int& c) {
  constexpr int GN = 8;
  const int g = t / (tiles_m * GN);
  const int gw = min(GN, tiles_n - g * GN);
  const int ti = t - g * tiles_m * GN;
  r = ti / gw;
  c = g * GN + ti % gw;
}

template <int BM, int BN, int WM, int WN>
__global__ __launch_bounds__(64 * WM * WN) void gemm_bf16_kernel(GemmArgs a) {
  constexpr int NT = 64 * WM * WN;  // threads per block
  constexpr int BK = 64;
  constexpr int LDK = BK + 8;  // +16 bytes per row: conflict-free 16-byte fragment reads
  constexpr int TM = BM / (16 * WM);
  constexpr int TN = BN / (16 * WN);
  constexpr int CA = BM * (BK / 8) / NT;  // 16-byte chunks per thread, A tile
  constexpr int CB = BN * (BK / 8) / NT;
  static_assert(CA >= 1 && CB >= 1, "tile too small");

  __shared__ __attribute__((aligned(16))) bf16_t As[2][BM][LDK];
  __shared__ __attribute__((aligned(16))) bf16_t Bs[2][BN][LDK];
  __shared__ int s_last;

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int l16 = lane & 15, grp = lane >> 4;
  const int wm = wave / WN, wn = wave % WN;

  const int tiles_n = (a.N + BN - 1) / BN;
  const int tile = xcd_tile(blockIdx.x, gridDim.x);
  int tr, tc;
  tile_rc(tile, gridDim.x / tiles_n, tiles_n, tr, tc);
  const int m0 = tr * BM;
  const int n0 = tc * BN;
  if (a.m_rows) a.M = min(a.M, *a.m_rows);
  if (m0 >= a.M) return;  // whole tile past a device-side row count (every K range alike)
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
      const int c = tid + i * NT;
      const int row = c >> 3, kc = (c & 7) * 8;
      const int m = m0 + row, k = k0 + kc;
      if (m < a.M && k < kend)
        ra[i] = *(const u32x4_t*)(A + (size_t)m * a.lda + k);
      else
        ra[i] = u32x4_t{0, 0, 0, 0};
    }
#pragma unroll
    for (int i = 0; i < CB; ++i) {
      const int c = tid + i * NT;
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
      const int c = tid + i * NT;
      *(u32x4_t*)&As[buf][c >> 3][(c & 7) * 8] = ra[i];
    }
#pragma unroll
    for (int i = 0; i < CB; ++i) {
      const int c = tid + i * NT;
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
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(bfr[j], af[i], acc[i][j], 0, 0, 0);
    }
    if (kt + 1 < nk) sstore(buf ^ 1);
    __syncthreads();
  }

  // acc[i][j][r] = C[m0 + wm*(BM/WM) + i*16 + l16][n0 + wn*(BN/WN) + j*16 + grp*4 + r]
  // (the weights are the MFMA's A operand, so each lane owns 4 consecutive columns)
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

  epilogue(a, acc, mw, nw, l16, grp);
}


// ---------------------------------------------------------------------------
// Tiled GEMM, many rows, K tiles loaded straight into LDS (global_load_lds,
// 16 bytes per lane): no register staging and no LDS store instructions.
// STAGES LDS buffers; tile kt + STAGES - 1 is in flight while tile kt is
// multiplied.  Rows are 64 bf16 (128 bytes, unpadded); the 16-byte chunk c of
// row r sits at chunk position c ^ ((r >> 1) & 7), so the 16 rows read by one
// fragment load hit 16 distinct bank groups.  Loads clamp rows to the matrix
// (rows / columns past M / N only feed outputs that are never written); K and
// the K range must be multiples of 64.  The fragment reads are inline asm with
// an explicit LDS wait: as plain loads the compiler would wait for every
// global->LDS load in flight (including later stages) before each of them, and
// __syncthreads() would wait for them too, so the K loop uses s_barrier after
// an explicit wait for this wave's loads of the current tile.
// ---------------------------------------------------------------------------
typedef __attribute__((address_space(3))) void lds_void_t;
typedef const __attribute__((address_space(1))) void gmem_void_t;

// gfx9 s_waitcnt immediate: vmcnt <= n, expcnt and lgkmcnt not waited for
constexpr unsigned waitcnt_vm(int n) { return (unsigned)((n & 0xF) | ((n >> 4) << 14) | (0x7 << 4) | (0xF << 8)); }

// ROWLOOP: the row count is known on the device only (a.m_rows); block b owns
// column tile b and runs every live row tile of it in turn (no K split, fp32
// output: EPI_F32 only).
// MODE: the epilogue, fixed at compile time (a run-time switch over the modes
// makes the compiler keep the accumulators in scratch memory).
template <int BM, int BN, int WM, int WN, int STAGES, int MODE, bool ROWLOOP = false>
__global__ __launch_bounds__(64 * WM * WN) void gemm_lds_kernel(GemmArgs a) {
  constexpr int NW = WM * WN;
  constexpr int BK = 64;
  constexpr int TM = BM / (16 * WM), TN = BN / (16 * WN);
  constexpr int LA = BM / 8 / NW, LB = BN / 8 / NW;  // 1 KB (8-row) segments per wave per tile
  static_assert(LA >= 1 && LB >= 1 && (BM / 8) % NW == 0 && (BN / 8) % NW == 0, "segments per wave");
  constexpr int AHEAD = STAGES - 1;
  static_assert(AHEAD >= 1 && AHEAD <= 3, "stages");
  __shared__ __attribute__((aligned(1024))) bf16_t As[STAGES][BM * BK];
  __shared__ __attribute__((aligned(1024))) bf16_t Bs[STAGES][BN * BK];
  __shared__ int s_last;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l16 = lane & 15, grp = lane >> 4;
  const int wm = wave / WN, wn = wave % WN;
  const int tiles_n = (a.N + BN - 1) / BN;
  int tile, m0, n0;
  if constexpr (ROWLOOP) {
    tile = blockIdx.x;
    m0 = 0;
    n0 = tile * BN;
    a.M = min(a.M, *a.m_rows);
  } else {
    tile = xcd_tile(blockIdx.x, gridDim.x);
    int tr, tc;
    tile_rc(tile, gridDim.x / tiles_n, tiles_n, tr, tc);
    m0 = tr * BM;
    n0 = tc * BN;
    if (a.m_rows) a.M = min(a.M, *a.m_rows);
  }
  if (m0 >= a.M) return;  // whole tile past a device-side row count (every K range alike)
  const int z = blockIdx.z;
  const int kbeg = z * a.kchunk;
  const int kend = min(a.K, kbeg + a.kchunk);
  const int nk = (kend - kbeg) / BK;
  const bf16_t* __restrict__ A = (const bf16_t*)a.A;
  const bf16_t* __restrict__ B = (const bf16_t*)a.B;

  const int srow = lane >> 3, spos = lane & 7;  // lane -> (row in segment, chunk position)
  auto issue = [&](int kt, int st) {
    const int k0 = kbeg + kt * BK;
#pragma unroll
    for (int i = 0; i < LA; ++i) {
      const int seg = wave * LA + i, row = seg * 8 + srow;
      const int m = min(m0 + row, a.M - 1);
      const int c = spos ^ ((row >> 1) & 7);
      __builtin_amdgcn_global_load_lds((gmem_void_t*)(A + (size_t)m * a.lda + k0 + c * 8), (lds_void_t*)&As[st][seg * 512],
                                       16, 0, 0);
    }
#pragma unroll
    for (int i = 0; i < LB; ++i) {
      const int seg = wave * LB + i, row = seg * 8 + srow;
      const int n = min(n0 + row, a.N - 1);
      const int c = spos ^ ((row >> 1) & 7);
      __builtin_amdgcn_global_load_lds((gmem_void_t*)(B + (size_t)n * a.ldb + k0 + c * 8), (lds_void_t*)&Bs[st][seg * 512],
                                       16, 0, 0);
    }
  };
  auto frag = [&](const bf16_t* base, int row, int c) -> bf16x8_t {
    const unsigned addr =
        (unsigned)(size_t)(const __attribute__((address_space(3))) bf16_t*)(&base[row * BK + ((c ^ ((row >> 1) & 7)) * 8)]);
    bf16x8_t v;
    asm volatile("ds_read_b128 %0, %1" : "=v"(v) : "v"(addr));
    return v;
  };

  for (;;) {  // once, or (ROWLOOP) once per live row tile
  f32x4_t acc[TM][TN];
#pragma unroll
  for (int i = 0; i < TM; ++i)
#pragma unroll
    for (int j = 0; j < TN; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int t = 0; t < AHEAD; ++t)
    if (t < nk) issue(t, t);
  for (int kt = 0; kt < nk; ++kt) {
    const int st = kt % STAGES;
    // this wave's loads of tile kt are complete once at most the later tiles'
    // loads are outstanding (vector memory operations complete in order)
    const int later = min(AHEAD - 1, nk - 1 - kt);
    if (later >= 2)
      __builtin_amdgcn_s_waitcnt(waitcnt_vm(2 * (LA + LB)));
    else if (later == 1)
      __builtin_amdgcn_s_waitcnt(waitcnt_vm(LA + LB));
    else
      __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));
    __builtin_amdgcn_s_barrier();  // every wave's part of tile kt is in LDS; tile kt-1's buffer is free
    if (kt + AHEAD < nk) issue(kt + AHEAD, (kt + AHEAD) % STAGES);
    const bf16_t* as = As[st];
    const bf16_t* bs = Bs[st];
#pragma unroll
    for (int ks = 0; ks < BK / 32; ++ks) {
      bf16x8_t af[TM], bfr[TN];
#pragma unroll
      for (int i = 0; i < TM; ++i) af[i] = frag(as, wm * (BM / WM) + i * 16 + l16, ks * 4 + grp);
#pragma unroll
      for (int j = 0; j < TN; ++j) bfr[j] = frag(bs, wn * (BN / WN) + j * 16 + l16, ks * 4 + grp);
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
#pragma unroll
      for (int i = 0; i < TM; ++i) asm volatile("" : "+v"(af[i]));
#pragma unroll
      for (int j = 0; j < TN; ++j) asm volatile("" : "+v"(bfr[j]));
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(bfr[j], af[i], acc[i][j], 0, 0, 0);
    }
  }

  const int mw = m0 + wm * (BM / WM);
  const int nw = n0 + wn * (BN / WN);
  if (a.ksplit > 1) {
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
  epi_frags<MODE>(a, acc, mw, nw, l16, grp);
  if constexpr (!ROWLOOP) break;
  m0 += BM;
  if (m0 >= a.M) break;
  // every wave's LDS reads of this tile completed before its MFMAs; the next
  // tile's loads may overwrite the stages once all waves are here
  __syncthreads();
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
  auto load_frag = [&](int tile, int c, int f) -> bf16x8_t {
    const int n = tile * (64 * NFR) + wave * (16 * NFR) + c * 16 + l16;
    const int k = kbeg + f * 32 + grp * 8;
    return (n < a.N && k < a.K) ? *(const bf16x8_t*)(B + (size_t)n * a.ldb + k) : bf16x8_t{};
  };
  auto load_w = [&](int tile) {
#pragma unroll
    for (int c = 0; c < NFR; ++c)
#pragma unroll
      for (int f = 0; f < NF; ++f) wfr[c][f] = load_frag(tile, c, f);
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
    // each weight fragment is reloaded with the next tile's as soon as its last
    // MFMA has read it: the next tile streams in during this tile's MFMAs and
    // epilogue, with no second register buffer
    const int next = tile + (int)gridDim.x;
    const bool more = next < tiles;
#pragma unroll
    for (int f = 0; f < NF; ++f) {
#pragma unroll
      for (int i = 0; i < MT; ++i) {
        const bf16x8_t xf = *(const bf16x8_t*)&As[i * 16 + l16][f * 32 + grp * 8];
#pragma unroll
        for (int c = 0; c < NFR; ++c)
          acc[c][i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wfr[c][f], xf, acc[c][i], 0, 0, 0);
      }
      if (more) {
#pragma unroll
        for (int c = 0; c < NFR; ++c) wfr[c][f] = load_frag(next, c, f);
      }
    }

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
    f32x4_t t[MT][NFR];
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
      for (int c = 0; c < NFR; ++c) t[i][c] = acc[c][i];
    epilogue(a, t, 0, nw, l16, grp);
  }
}

template <int MT, int NFR, int KR>
static hipError_t launch_skinny_t(const GemmArgs& a, hipStream_t s) {
  const int tiles = (a.N + 64 * NFR - 1) / (64 * NFR);
  // one resident round of blocks (the row tile in LDS decides how many fit on a
  // CU); extra tiles are looped over inside a block, with their weights pipelined
  static int cus = 0;
  if (cus == 0) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
      cus = 256;
  }
  constexpr int lds_bytes = MT * 16 * (KR + 8) * 2;
  constexpr int per_cu = lds_bytes > 80 * 1024 ? 1 : 2;
  const int cap = (a.ksplit > 1) ? tiles : std::max(1, std::min(tiles, per_cu * cus));
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


// ---------------------------------------------------------------------------
// Register-streaming kernel for few rows (M <= 64) and a moderate number of
// columns.  Block = NW waves = one 64-column tile x all M rows x a K range of
// 64*NW.  Wave w takes its own 64-wide K slice for all 64 columns: its weight
// fragments (4 column blocks x 2 k-steps) and activation fragments (MT row
// blocks x 2 k-steps) are all loaded straight into registers at once, so a
// block pays one memory latency.  The NW partial tiles are summed through LDS
// in fixed wave order; K ranges of several blocks (grid.y) are reduced by the
// last-arriving block in fixed order.
// ---------------------------------------------------------------------------
template <int MT, int NW>
__global__ __launch_bounds__(64 * NW) void gemm_regstream_kernel(GemmArgs a) {
  constexpr int NC = 4;           // 16-column blocks per tile
  constexpr int FR = NC * MT;     // accumulator fragments per wave
  constexpr int KR = 64 * NW;     // K range of the block
  __shared__ __attribute__((aligned(16))) float red[NW][FR][64][4];
  __shared__ int s_last;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l16 = lane & 15, grp = lane >> 4;
  const int tile = blockIdx.x, z = blockIdx.y;
  const int n0 = tile * 64;
  const int kw = z * KR + wave * 64;  // this wave's K slice
  const bf16_t* __restrict__ A = (const bf16_t*)a.A;
  const bf16_t* __restrict__ B = (const bf16_t*)a.B;

  // buffer loads: a lane with nothing to load passes an offset past the
  // resource's range and reads zeros, so every load is issued unconditionally
  // and all of them are in flight together
  const __amdgpu_buffer_rsrc_t rA = __builtin_amdgcn_make_buffer_rsrc(const_cast<bf16_t*>(A), (short)0, 0x7fffffff,
                                                                       0x00020000);
  const __amdgpu_buffer_rsrc_t rB = __builtin_amdgcn_make_buffer_rsrc(const_cast<bf16_t*>(B), (short)0, 0x7fffffff,
                                                                       0x00020000);
  constexpr int kOOR = (int)0x80000000u;
  bf16x8_t wf[NC][2], xf[MT][2];
#pragma unroll
  for (int f = 0; f < 2; ++f) {
    const int k = kw + f * 32 + grp * 8;
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      const int n = n0 + c * 16 + l16;
      const int off = (n < a.N && k < a.K) ? (int)(((size_t)n * a.ldb + k) * 2) : kOOR;
      wf[c][f] = __builtin_bit_cast(bf16x8_t, __builtin_amdgcn_raw_buffer_load_b128(rB, off, 0, 0));
    }
#pragma unroll
    for (int i = 0; i < MT; ++i) {
      const int m = i * 16 + l16;
      const int off = (m < a.M && k < a.K) ? (int)(((size_t)m * a.lda + k) * 2) : kOOR;
      xf[i][f] = __builtin_bit_cast(bf16x8_t, __builtin_amdgcn_raw_buffer_load_b128(rA, off, 0, 0));
    }
  }
  f32x4_t acc[NC][MT];
#pragma unroll
  for (int c = 0; c < NC; ++c)
#pragma unroll
    for (int i = 0; i < MT; ++i) {
      acc[c][i] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int f = 0; f < 2; ++f)
        acc[c][i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wf[c][f], xf[i][f], acc[c][i], 0, 0, 0);
    }
#pragma unroll
  for (int c = 0; c < NC; ++c)
#pragma unroll
    for (int i = 0; i < MT; ++i) *(f32x4_t*)&red[wave][c * MT + i][lane][0] = acc[c][i];
  __syncthreads();

  // sum the waves' partial tiles in fixed order: item = (fragment, lane)
  constexpr int ITEMS = FR * 64;
  constexpr int PER = (ITEMS + 64 * NW - 1) / (64 * NW);
  f32x4_t sum[PER];
#pragma unroll
  for (int q = 0; q < PER; ++q) {
    const int item = tid + q * 64 * NW;
    sum[q] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    if (item < ITEMS) {
#pragma unroll
      for (int w = 0; w < NW; ++w) {
        const f32x4_t v = *(const f32x4_t*)&red[w][item >> 6][item & 63][0];
        sum[q][0] += v[0];
        sum[q][1] += v[1];
        sum[q][2] += v[2];
        sum[q][3] += v[3];
      }
    }
  }

  if (a.ksplit > 1) {
    const size_t tile_elems = (size_t)ITEMS * 4;
    float* part = a.partial + ((size_t)z * gridDim.x + tile) * tile_elems;
#pragma unroll
    for (int q = 0; q < PER; ++q) {
      const int item = tid + q * 64 * NW;
      if (item < ITEMS) coherent_store4(part + (size_t)item * 4, sum[q]);
    }
    if (!last_block_arrival(&a.counters[tile * kCounterStride], (unsigned)a.ksplit, &s_last)) return;
#pragma unroll
    for (int q = 0; q < PER; ++q) {
      const int item = tid + q * 64 * NW;
      if (item >= ITEMS) continue;
      f32x4_t t = {0.f, 0.f, 0.f, 0.f};
      for (int zz = 0; zz < a.ksplit; ++zz) {
        const f32x4_t v = (zz == z) ? sum[q]
                                    : *(const f32x4_t*)(a.partial + ((size_t)zz * gridDim.x + tile) * tile_elems +
                                                        (size_t)item * 4);
        t[0] += v[0];
        t[1] += v[1];
        t[2] += v[2];
        t[3] += v[3];
      }
      sum[q] = t;
    }
  }

  // item = (c * MT + i) * 64 + lane: rows i*16 + (lane & 15), columns n0 + c*16 + 4*(lane >> 4)
  if (a.mode == EPI_GEGLU) {
    // gate block c (even) and up block c + 1 are items (c*MT+i)*64+lane and ((c+1)*MT+i)*64+lane;
    // route both to the thread owning the gate item through LDS
    __syncthreads();
#pragma unroll
    for (int q = 0; q < PER; ++q) {
      const int item = tid + q * 64 * NW;
      if (item < ITEMS) *(f32x4_t*)&red[0][item >> 6][item & 63][0] = sum[q];
    }
    __syncthreads();
#pragma unroll
    for (int q = 0; q < PER; ++q) {
      const int item = tid + q * 64 * NW;
      if (item >= ITEMS) continue;
      const int fr = item >> 6, ln = item & 63;
      const int c = fr / MT, i = fr % MT;
      if (c & 1) continue;
      const int m = i * 16 + (ln & 15);
      const int ng = n0 + c * 16;
      if (m < a.M && ng < a.N) {
        const f32x4_t u = *(const f32x4_t*)&red[0][(c + 1) * MT + i][ln][0];
        epi_geglu4(a, m, (ng >> 5) * 16 + (ln >> 4) * 4, sum[q], u);
      }
    }
    return;
  }
  const bool vec = epi_vec_ok(a);
#pragma unroll
  for (int q = 0; q < PER; ++q) {
    const int item = tid + q * 64 * NW;
    if (item >= ITEMS) continue;
    const int fr = item >> 6, ln = item & 63;
    const int c = fr / MT, i = fr % MT;
    const int m = i * 16 + (ln & 15), n = n0 + c * 16 + (ln >> 4) * 4;
    if (m >= a.M || n >= a.N) continue;
    switch (a.mode) {
      case EPI_F32: epi4<EPI_F32>(a, m, n, sum[q], vec); break;
      case EPI_T: epi4<EPI_T>(a, m, n, sum[q], vec); break;
      case EPI_RESID: epi4<EPI_RESID>(a, m, n, sum[q], vec); break;
      case EPI_RESID_TANH: epi4<EPI_RESID_TANH>(a, m, n, sum[q], vec); break;
      case EPI_COND: epi4<EPI_COND>(a, m, n, sum[q], vec); break;
      case EPI_GELU_T: epi4<EPI_GELU_T>(a, m, n, sum[q], vec); break;
      case EPI_SILU_T: epi4<EPI_SILU_T>(a, m, n, sum[q], vec); break;
      default: break;
    }
  }
}

// ---------------------------------------------------------------------------
// Whole-K kernel for few rows (M <= 64) and K <= 1024 (K % 128 == 0): block = 32
// output columns x all M rows x the whole K; wave w takes the K quarter
// [w K/4, (w + 1) K/4) and loads all its weight and activation fragments at once.
// The four partial tiles are added through LDS in fixed wave order, so no K range
// is split across blocks: no partial tiles, no tickets, one memory latency.
// ---------------------------------------------------------------------------
// The first adaptive norm's operands from modulation values v (columns n .. n+3 of
// row m, see GemmArgs::nrm_p).
RAVEL_DEV void norm_operands4(const GemmArgs& a, int m, int n, f32x4_t v) {
  const int w = a.nrm_w;
  const auto t32 = [](int row, int c) { return ((size_t)(c >> 5) * 64 + row) * 32 + (c & 31); };
  if (n < w) {
    const f32x4_t x = *(const f32x4_t*)(a.nrm_x + (size_t)m * w + n);
    u32x2_t o;
    o[0] = (uint32_t)f32_to_bf16((1.f + v[0]) * x[0]) | ((uint32_t)f32_to_bf16((1.f + v[1]) * x[1]) << 16);
    o[1] = (uint32_t)f32_to_bf16((1.f + v[2]) * x[2]) | ((uint32_t)f32_to_bf16((1.f + v[3]) * x[3]) << 16);
    *(u32x2_t*)(a.nrm_p + t32(m, n)) = o;
    return;
  }
  const int c = (n >= w && n < 2 * w) ? 0 : ((n >= 4 * w && n < 5 * w) ? 1 : -1);
  if (c < 0) return;
  const int col = n - (c == 0 ? w : 4 * w);
  const u32x2_t o = {pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3])};
  *(u32x2_t*)(a.nrm_shift + (size_t)c * 64 * w + t32(m, col)) = o;
}

// block bx of a whole-K launch (32 output columns)
template <int MT>
RAVEL_DEV void gemm_wholek_block(const GemmArgs& a, int bx) {
  constexpr int NC = 2;            // 16-column blocks per block
  constexpr int FR = NC * MT;      // accumulator fragments per wave
  __shared__ __attribute__((aligned(16))) float red[4][FR][64][4];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l16 = lane & 15, grp = lane >> 4;
  const int n0 = bx * 32;
  const int kq = a.K >> 2, kb = wave * kq;  // kq: a multiple of 32, at most 256
  const bf16_t* __restrict__ A = (const bf16_t*)a.A;
  const bf16_t* __restrict__ B = (const bf16_t*)a.B;
  const __amdgpu_buffer_rsrc_t rA = __builtin_amdgcn_make_buffer_rsrc(const_cast<bf16_t*>(A), (short)0, 0x7fffffff,
                                                                       0x00020000);
  const __amdgpu_buffer_rsrc_t rB = __builtin_amdgcn_make_buffer_rsrc(const_cast<bf16_t*>(B), (short)0, 0x7fffffff,
                                                                       0x00020000);
  constexpr int kOOR = (int)0x80000000u;
  // fragments past the wave's K quarter, rows past M and columns past N read zeros
  bf16x8_t wf[NC][8], xf[MT][8];
#pragma unroll
  for (int f = 0; f < 8; ++f) {
    const int k = kb + f * 32 + grp * 8;
    const bool kin = f * 32 < kq;
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      const int n = n0 + c * 16 + l16;
      const int off = (kin && n < a.N) ? (int)(((size_t)n * a.ldb + k) * 2) : kOOR;
      wf[c][f] = __builtin_bit_cast(bf16x8_t, __builtin_amdgcn_raw_buffer_load_b128(rB, off, 0, 0));
    }
  }
#pragma unroll
  for (int f = 0; f < 8; ++f) {
    const int k = kb + f * 32 + grp * 8;
    const bool kin = f * 32 < kq;
#pragma unroll
    for (int i = 0; i < MT; ++i) {
      const int m = i * 16 + l16;
      const int off = (kin && m < a.M) ? (int)(((size_t)m * a.lda + k) * 2) : kOOR;
      xf[i][f] = __builtin_bit_cast(bf16x8_t, __builtin_amdgcn_raw_buffer_load_b128(rA, off, 0, 0));
    }
  }
  f32x4_t acc[NC][MT];
#pragma unroll
  for (int c = 0; c < NC; ++c)
#pragma unroll
    for (int i = 0; i < MT; ++i) {
      acc[c][i] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int f = 0; f < 8; ++f)
        acc[c][i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wf[c][f], xf[i][f], acc[c][i], 0, 0, 0);
    }
#pragma unroll
  for (int c = 0; c < NC; ++c)
#pragma unroll
    for (int i = 0; i < MT; ++i) *(f32x4_t*)&red[wave][c * MT + i][lane][0] = acc[c][i];
  __syncthreads();
  // item = (c * MT + i) * 64 + lane: rows i*16 + (lane & 15), columns n0 + c*16 + 4*(lane >> 4)
  const bool vec = epi_vec_ok(a);
  for (int item = tid; item < FR * 64; item += 256) {
    const int fr = item >> 6, ln = item & 63;
    const int c = fr / MT, i = fr % MT;
    f32x4_t s = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const f32x4_t v = *(const f32x4_t*)&red[w][fr][ln][0];
      s[0] += v[0];
      s[1] += v[1];
      s[2] += v[2];
      s[3] += v[3];
    }
    const int m = i * 16 + (ln & 15), n = n0 + c * 16 + (ln >> 4) * 4;
    if (m >= a.M || n >= a.N) continue;
    if (a.nrm_p && a.mode == EPI_F32 && n + 4 <= a.N) {
      const f32x4_t b4 = a.bias ? *(const f32x4_t*)(a.bias + n) : f32x4_t{0.f, 0.f, 0.f, 0.f};
      norm_operands4(a, m, n, f32x4_t{s[0] + b4[0], s[1] + b4[1], s[2] + b4[2], s[3] + b4[3]});
    }
    switch (a.mode) {
      case EPI_F32: epi4<EPI_F32>(a, m, n, s, vec); break;
      case EPI_T: epi4<EPI_T>(a, m, n, s, vec); break;
      case EPI_RESID: epi4<EPI_RESID>(a, m, n, s, vec); break;
      case EPI_RESID_TANH: epi4<EPI_RESID_TANH>(a, m, n, s, vec); break;
      case EPI_COND: epi4<EPI_COND>(a, m, n, s, vec); break;
      case EPI_GELU_T: epi4<EPI_GELU_T>(a, m, n, s, vec); break;
      case EPI_SILU_T: epi4<EPI_SILU_T>(a, m, n, s, vec); break;
      default: break;
    }
  }
}

template <int MT>
__global__ __launch_bounds__(256) void gemm_wholek_kernel(GemmArgs a) {
  gemm_wholek_block<MT>(a, blockIdx.x);
}

// two GEMMs: blocks [0, nb1) take a1, the rest a2
template <int MT1, int MT2>
__global__ __launch_bounds__(256) void gemm_wholek2_kernel(GemmArgs a1, int nb1, GemmArgs a2) {
  if ((int)blockIdx.x < nb1)
    gemm_wholek_block<MT1>(a1, blockIdx.x);
  else
    gemm_wholek_block<MT2>(a2, blockIdx.x - nb1);
}

template <int MT>
static hipError_t launch_wholek_t(const GemmArgs& a, hipStream_t s) {
  hipLaunchKernelGGL((gemm_wholek_kernel<MT>), dim3((a.N + 31) / 32), dim3(256), 0, s, a);
  return hipGetLastError();
}

template <int MT, int NW>
static hipError_t launch_regstream_t(const GemmArgs& a, hipStream_t s) {
  dim3 grid((a.N + 63) / 64, a.ksplit);
  hipLaunchKernelGGL((gemm_regstream_kernel<MT, NW>), grid, dim3(64 * NW), 0, s, a);
  return hipGetLastError();
}

template <int MT>
static hipError_t launch_regstream_m(const GemmArgs& a, hipStream_t s) {
  switch (a.kchunk) {
    case 256: return launch_regstream_t<MT, 4>(a, s);
    case 512: return launch_regstream_t<MT, 8>(a, s);
    default: return hipErrorInvalidValue;
  }
}

// operands addressed through buffer resources with 32-bit byte offsets
static bool fits_buffer(const GemmArgs& a) {
  return (size_t)a.N * a.ldb * 2 < 0x7fffffffull && (size_t)a.M * a.lda * 2 < 0x7fffffffull;
}

hipError_t launch_gemm_regstream(const GemmArgs& a, hipStream_t s) {
  if (a.M > 64 || (a.mode == EPI_GEGLU && a.N % 32)) return hipErrorInvalidValue;
  if (a.ksplit * a.kchunk < a.K || !fits_buffer(a)) return hipErrorInvalidValue;
  switch ((a.M + 15) / 16) {
    case 1: return launch_regstream_m<1>(a, s);
    case 2: return launch_regstream_m<2>(a, s);
    case 3: return launch_regstream_m<3>(a, s);
    default: return launch_regstream_m<4>(a, s);
  }
}

static bool wholek_ok(const GemmArgs& a) {
  if (a.M > 64 || a.K > 1024 || (a.K % 128) || a.mode == EPI_GEGLU || !fits_buffer(a)) return false;
  // the norm operands: modulation rows of 6 nrm_w columns, 4-column groups inside one chunk
  if (a.nrm_p && (a.mode != EPI_F32 || !a.nrm_x || !a.nrm_shift || a.nrm_w % 32 || a.N != 6 * a.nrm_w)) return false;
  return true;
}

hipError_t launch_gemm_wholek2(const GemmArgs& a1, const GemmArgs& a2, hipStream_t s) {
  if (!wholek_ok(a1) || !wholek_ok(a2)) return hipErrorInvalidValue;
  // the pairs used: a few rows' modulation (4 row fragments) with the FOP tokens' keys
  // and values (1 row fragment)
  if ((a1.M + 15) / 16 != 4 || (a2.M + 15) / 16 != 1) return hipErrorInvalidValue;
  const int nb1 = (a1.N + 31) / 32, nb2 = (a2.N + 31) / 32;
  hipLaunchKernelGGL((gemm_wholek2_kernel<4, 1>), dim3(nb1 + nb2), dim3(256), 0, s, a1, nb1, a2);
  return hipGetLastError();
}

hipError_t launch_gemm_wholek(const GemmArgs& a, hipStream_t s) {
  if (!wholek_ok(a)) return hipErrorInvalidValue;
  switch ((a.M + 15) / 16) {
    case 1: return launch_wholek_t<1>(a, s);
    case 2: return launch_wholek_t<2>(a, s);
    case 3: return launch_wholek_t<3>(a, s);
    default: return launch_wholek_t<4>(a, s);
  }
}

template <int BM, int BN, int WM, int WN>
static hipError_t launch_tile(const GemmArgs& a, hipStream_t s) {
  const int tiles = ((a.M + BM - 1) / BM) * ((a.N + BN - 1) / BN);
  dim3 grid(tiles, 1, a.ksplit);
  hipLaunchKernelGGL((gemm_bf16_kernel<BM, BN, WM, WN>), grid, dim3(64 * WM * WN), 0, s, a);
  return hipGetLastError();
}

template <int BM, int BN, int WM, int WN, int STAGES, int MODE>
static hipError_t launch_lds_tile_m(const GemmArgs& a, hipStream_t s) {
  const int tiles = ((a.M + BM - 1) / BM) * ((a.N + BN - 1) / BN);
  dim3 grid(tiles, 1, a.ksplit);
  hipLaunchKernelGGL((gemm_lds_kernel<BM, BN, WM, WN, STAGES, MODE>), grid, dim3(64 * WM * WN), 0, s, a);
  return hipGetLastError();
}

template <int BM, int BN, int WM, int WN, int STAGES>
static hipError_t launch_lds_tile(const GemmArgs& a, hipStream_t s) {
  switch (a.mode) {
    case EPI_F32: return launch_lds_tile_m<BM, BN, WM, WN, STAGES, EPI_F32>(a, s);
    case EPI_T: return launch_lds_tile_m<BM, BN, WM, WN, STAGES, EPI_T>(a, s);
    case EPI_RESID: return launch_lds_tile_m<BM, BN, WM, WN, STAGES, EPI_RESID>(a, s);
    case EPI_RESID_TANH: return launch_lds_tile_m<BM, BN, WM, WN, STAGES, EPI_RESID_TANH>(a, s);
    case EPI_GEGLU: return launch_lds_tile_m<BM, BN, WM, WN, STAGES, EPI_GEGLU>(a, s);
    case EPI_COND: return launch_lds_tile_m<BM, BN, WM, WN, STAGES, EPI_COND>(a, s);
    case EPI_GELU_T: return launch_lds_tile_m<BM, BN, WM, WN, STAGES, EPI_GELU_T>(a, s);
    case EPI_SILU_T: return launch_lds_tile_m<BM, BN, WM, WN, STAGES, EPI_SILU_T>(a, s);
    default: return hipErrorInvalidValue;
  }
}

// row-loop launches (device-side row count) have the fp32 epilogue only
template <int BM, int BN, int WM, int WN, int STAGES>
static hipError_t launch_lds_rows(const GemmArgs& a, hipStream_t s) {
  hipLaunchKernelGGL((gemm_lds_kernel<BM, BN, WM, WN, STAGES, EPI_F32, true>), dim3((a.N + BN - 1) / BN),
                     dim3(64 * WM * WN), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_gemm_bf16(const GemmArgs& a, int tile, hipStream_t s) {
  // direct-to-LDS variants (measured on MI355X at M = 3200: 128x128 with two
  // stages 744-804 TF/s at K = 1024; 128x64 with three stages 514-581 TF/s at
  // N = 1024, K = 2048-4096) where K tiles are whole and rows 16-byte aligned
  const bool lds_ok = a.K % 64 == 0 && a.kchunk % 64 == 0 && a.lda % 8 == 0 && a.ldb % 8 == 0 &&
                      ((uintptr_t)a.A % 16) == 0 && ((uintptr_t)a.B % 16) == 0 && a.M > 0 && a.N > 0;
  // device-side row count (few distinct rows, many columns): 256-row tiles, one
  // block per column tile, so every weight byte is streamed once
  if (lds_ok && a.m_rows && a.ksplit == 1 && a.mode == EPI_F32) return launch_lds_rows<256, 128, 4, 2, 2>(a, s);
  if (lds_ok && tile == TILE_128x128) return launch_lds_tile<128, 128, 2, 2, 2>(a, s);
  if (lds_ok && tile == TILE_128x64) return launch_lds_tile<128, 64, 2, 2, 3>(a, s);
  // larger wave tiles (64x128 .. 128x128) read less LDS per MFMA flop
  if (lds_ok && tile == TILE_128x256) return launch_lds_tile<128, 256, 2, 2, 2>(a, s);
  if (lds_ok && tile == TILE_256x128) return launch_lds_tile<256, 128, 2, 2, 2>(a, s);
  if (lds_ok && tile == TILE_256x256) return launch_lds_tile<256, 256, 2, 2, 2>(a, s);
  switch (tile) {
    case TILE_128x128: return launch_tile<128, 128, 2, 2>(a, s);
    case TILE_64x128: return launch_tile<64, 128, 2, 2>(a, s);
    case TILE_128x64: return launch_tile<128, 64, 2, 2>(a, s);
    case TILE_32x64: return launch_tile<32, 64, 1, 4>(a, s);
    case TILE_256x128: return launch_tile<256, 128, 2, 2>(a, s);
    case TILE_128x256: return launch_tile<128, 256, 2, 2>(a, s);
    case TILE_256x256: return launch_tile<256, 256, 4, 2>(a, s);
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
  if (a.m_rows) a.M = min(a.M, *a.m_rows);
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
    ((float*)a.out_t)[(size_t)m * a.ldo_t + n] = gelu_tanh_f(g) * u;
  } else {
    if (n >= a.N) return;
    const float* b = B + (size_t)n * a.ldb;
    float acc = 0.f;
    for (int k = 0; k < a.K; ++k) acc += A[k] * b[k];
    switch (a.mode) {
      case EPI_F32: epi1<EPI_F32, float>(a, m, n, acc); break;
      case EPI_T: epi1<EPI_T, float>(a, m, n, acc); break;
      case EPI_RESID: epi1<EPI_RESID, float>(a, m, n, acc); break;
      case EPI_RESID_TANH: epi1<EPI_RESID_TANH, float>(a, m, n, acc); break;
      case EPI_COND: epi1<EPI_COND, float>(a, m, n, acc); break;
      case EPI_GELU_T: epi1<EPI_GELU_T, float>(a, m, n, acc); break;
      case EPI_SILU_T: epi1<EPI_SILU_T, float>(a, m, n, acc); break;
      default: break;
    }
  }
}

hipError_t launch_gemm_f32(const GemmArgs& a, hipStream_t s) {
  const int ncols = a.mode == EPI_GEGLU ? a.N / 2 : a.N;
  dim3 grid((ncols + 63) / 64, (a.M + 3) / 4);
  hipLaunchKernelGGL(gemm_f32_kernel, grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

}  // namespace ravel
