// Row and element-wise kernels of the rolling step: adaptive RMSNorm (one
// wavefront per row), offset conditioning, input projection in logical slot
// order, analytic velocity fields, the fused Euler / release / Philox-append
// kernel, ring initialisation, the flow-time embedding and small utilities.
#include "kernels.h"

namespace ravel {

// ---------------------------------------------------------------------------
// Philox4x32-10 (Salmon, Moraes, Dror, Shaw, SC'11) and Box-Muller.
// ---------------------------------------------------------------------------
RAVEL_DEV void philox4x32_10(uint32_t c[4], uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    if (r > 0) {
      k0 += 0x9E3779B9u;
      k1 += 0xBB67AE85u;
    }
    const uint32_t lo0 = 0xD2511F53u * c[0];
    const uint32_t hi0 = __umulhi(0xD2511F53u, c[0]);
    const uint32_t lo1 = 0xCD9E8D57u * c[2];
    const uint32_t hi1 = __umulhi(0xCD9E8D57u, c[2]);
    const uint32_t n0 = hi1 ^ c[1] ^ k0;
    const uint32_t n2 = hi0 ^ c[3] ^ k1;
    c[0] = n0;
    c[1] = lo1;
    c[2] = n2;
    c[3] = lo0;
  }
}

// Two normals from a (radius word, angle word) pair: float64, rounded to float32.
RAVEL_DEV void box_muller(uint32_t xr, uint32_t xa, float* z0, float* z1) {
  const double ua = ((double)(xr >> 8) + 1.0) * 5.9604644775390625e-08;  // 2^-24
  const double ub = (double)(xa >> 8) * 5.9604644775390625e-08;
  const double rad = sqrt(-2.0 * log(ua));
  const double ang = 6.283185307179586 * ub;
  *z0 = (float)(rad * cos(ang));
  *z1 = (float)(rad * sin(ang));
}

// Noise of action r for env e, elements 4c .. 4c+3.
RAVEL_DEV void ring_noise4(uint64_t seed, int e, int64_t r, int c, float z[4]) {
  uint32_t ctr[4] = {(uint32_t)c, (uint32_t)e, (uint32_t)((uint64_t)r & 0xFFFFFFFFu),
                     (uint32_t)((uint64_t)r >> 32)};
  philox4x32_10(ctr, (uint32_t)(seed & 0xFFFFFFFFu), (uint32_t)(seed >> 32));
  box_muller(ctr[0], ctr[1], &z[0], &z[1]);
  box_muller(ctr[2], ctr[3], &z[2], &z[3]);
}

// ---------------------------------------------------------------------------
// Adaptive RMSNorm
// ---------------------------------------------------------------------------
template <typename T>
RAVEL_DEV void store4(T* p, float v0, float v1, float v2, float v3);
template <>
RAVEL_DEV void store4<float>(float* p, float v0, float v1, float v2, float v3) {
  *(f32x4_t*)p = f32x4_t{v0, v1, v2, v3};
}
template <>
RAVEL_DEV void store4<bf16_t>(bf16_t* p, float v0, float v1, float v2, float v3) {
  *(u32x2_t*)p = u32x2_t{pack_bf16x2(v0, v1), pack_bf16x2(v2, v3)};
}

// One wavefront per row, 4 consecutive features per lane and access.  For
// w <= 256 * NCH the row stays in registers: the row, its modulation-row index
// and (once that is known) its scale and shift are all requested before the
// reduction, so a row costs two memory round trips.  NCH = 0: any width, the
// row is read twice.
template <typename T, int NCH>
__global__ __launch_bounds__(256) void adarms_kernel(const float* __restrict__ x, int ldx, int M, int w,
                                                     const float* __restrict__ scale,
                                                     const float* __restrict__ shift, int ldm, int mode,
                                                     const int* __restrict__ rowmap, float eps,
                                                     T* __restrict__ y, int ldy) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= M) return;
  const float* xr = x + (size_t)row * ldx;
  T* yr = y + (size_t)row * ldy;
  if constexpr (NCH > 0) {
    const size_t mrow = rowmap ? (size_t)rowmap[row] : (size_t)row;
    f32x4_t v[NCH], sc[NCH], sh[NCH];
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      const int n = lane * 4 + c * 256;
      v[c] = n < w ? *(const f32x4_t*)(xr + n) : f32x4_t{0.f, 0.f, 0.f, 0.f};
    }
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      const int n = lane * 4 + c * 256;
      const f32x4_t z = {0.f, 0.f, 0.f, 0.f};
      sc[c] = n < w ? *(const f32x4_t*)(scale + (mode == 0 ? mrow * ldm : 0) + n) : z;
      sh[c] = (n < w && mode == 0) ? *(const f32x4_t*)(shift + mrow * ldm + n) : z;
    }
    float ss = 0.f;
#pragma unroll
    for (int c = 0; c < NCH; ++c) ss += v[c][0] * v[c][0] + v[c][1] * v[c][1] + v[c][2] * v[c][2] + v[c][3] * v[c][3];
    ss = wave_sum(ss);
    const float r = 1.0f / sqrtf(ss / (float)w + eps);
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      const int n = lane * 4 + c * 256;
      if (n >= w) continue;
      float o[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) o[i] = v[c][i] * r * (1.0f + sc[c][i]) + sh[c][i];
      store4<T>(yr + n, o[0], o[1], o[2], o[3]);
    }
    return;
  }
  float ss = 0.f;
  for (int n = lane * 4; n < w; n += 256) {
    const f32x4_t v = *(const f32x4_t*)(xr + n);
    ss += v[0] * v[0] + v[1] * v[1] + v[2] * v[2] + v[3] * v[3];
  }
  ss = wave_sum(ss);
  const float r = 1.0f / sqrtf(ss / (float)w + eps);
  const size_t mrow = rowmap ? (size_t)rowmap[row] : (size_t)row;
  for (int n = lane * 4; n < w; n += 256) {
    const f32x4_t v = *(const f32x4_t*)(xr + n);
    float o[4];
    if (mode == 0) {
      const f32x4_t sc = *(const f32x4_t*)(scale + mrow * ldm + n);
      const f32x4_t sh = *(const f32x4_t*)(shift + mrow * ldm + n);
#pragma unroll
      for (int i = 0; i < 4; ++i) o[i] = v[i] * r * (1.0f + sc[i]) + sh[i];
    } else {
      const f32x4_t sc = *(const f32x4_t*)(scale + n);
#pragma unroll
      for (int i = 0; i < 4; ++i) o[i] = v[i] * r * (1.0f + sc[i]);
    }
    store4<T>(yr + n, o[0], o[1], o[2], o[3]);
  }
}

template <typename T>
hipError_t launch_adarms(const float* x, int ldx, int M, int w, const float* scale, const float* shift,
                         int ldm, int mode, const int* rowmap, float eps, T* y, int ldy, hipStream_t s) {
  // 16-byte accesses: w, the row strides and the base pointers must be multiples of 4 floats
  if (w % 4 || ldx % 4 || ldy % 4 || (mode == 0 && ldm % 4) || ((uintptr_t)x | (uintptr_t)scale) % 16 ||
      (mode == 0 && (uintptr_t)shift % 16) || (uintptr_t)y % (4 * sizeof(T)))
    return hipErrorInvalidValue;
  const dim3 grid((M + 3) / 4), block(256);
  if (w <= 256)
    hipLaunchKernelGGL((adarms_kernel<T, 1>), grid, block, 0, s, x, ldx, M, w, scale, shift, ldm, mode, rowmap, eps, y, ldy);
  else if (w <= 512)
    hipLaunchKernelGGL((adarms_kernel<T, 2>), grid, block, 0, s, x, ldx, M, w, scale, shift, ldm, mode, rowmap, eps, y, ldy);
  else if (w <= 1024)
    hipLaunchKernelGGL((adarms_kernel<T, 4>), grid, block, 0, s, x, ldx, M, w, scale, shift, ldm, mode, rowmap, eps, y, ldy);
  else if (w <= 2048)
    hipLaunchKernelGGL((adarms_kernel<T, 8>), grid, block, 0, s, x, ldx, M, w, scale, shift, ldm, mode, rowmap, eps, y, ldy);
  else
    hipLaunchKernelGGL((adarms_kernel<T, 0>), grid, block, 0, s, x, ldx, M, w, scale, shift, ldm, mode, rowmap, eps, y, ldy);
  return hipGetLastError();
}
template hipError_t launch_adarms<float>(const float*, int, int, int, const float*, const float*, int, int,
                                         const int*, float, float*, int, hipStream_t);
template hipError_t launch_adarms<bf16_t>(const float*, int, int, int, const float*, const float*, int,
                                          int, const int*, float, bf16_t*, int, hipStream_t);

// ---------------------------------------------------------------------------
// Conditioning groups: envs with equal t_obs share delta, hence cond and every
// modulation row, within a step.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(256) void cond_groups_kernel(const int64_t* __restrict__ t_obs, int B, int H,
                                                          int* __restrict__ grp, int* __restrict__ rowmap,
                                                          int* __restrict__ rows) {
  __shared__ int64_t to[kCondGroupsMaxB];
  __shared__ int first[kCondGroupsMaxB];  // first env with the same t_obs
  __shared__ int rank[kCondGroupsMaxB];   // group index of a first env
  const int tid = threadIdx.x;
  for (int e = tid; e < B; e += 256) to[e] = t_obs[e];
  __syncthreads();
  for (int e = tid; e < B; e += 256) {
    int f = e;
    for (int j = 0; j < e; ++j)
      if (to[j] == to[e]) {
        f = j;
        break;
      }
    first[e] = f;
  }
  __syncthreads();
  for (int e = tid; e < B; e += 256) {
    if (first[e] != e) continue;
    int c = 0;
    for (int j = 0; j < e; ++j) c += first[j] == j;
    rank[e] = c;
  }
  __syncthreads();
  for (int e = tid; e < B; e += 256) {
    const int g = rank[first[e]];
    grp[e] = first[e] == e ? g : -1 - g;
  }
  for (int m = tid; m < B * H; m += 256) rowmap[m] = rank[first[m / H]] * H + m % H;
  if (tid == 0) {
    int n = 0;
    for (int e = 0; e < B; ++e) n += first[e] == e;
    rows[0] = n * H;
  }
}

hipError_t launch_cond_groups(const int64_t* t_obs, int B, int H, int* grp, int* rowmap, int* rows,
                              hipStream_t s) {
  if (B < 1 || B > kCondGroupsMaxB || H < 1) return hipErrorInvalidValue;
  hipLaunchKernelGGL(cond_groups_kernel, dim3(1), dim3(256), 0, s, t_obs, B, H, grp, rowmap, rows);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Offset conditioning hidden layer
// ---------------------------------------------------------------------------
template <typename T>
__global__ void delta_hidden_kernel(const int64_t* t, const int64_t* t_obs, const int64_t* ages, int B, int H,
                                    float delta_bias, const float* wd1, const float* bd1, int w, T* h1) {
  const int e = blockIdx.y;
  const int n = blockIdx.x * blockDim.x + threadIdx.x;
  if (n >= w || e >= B) return;
  // context age: given per env, or t - t_obs, or 0 without a step counter
  const float p = ages ? (float)ages[e] : (t ? (float)(*t - t_obs[e]) : 0.f);
  const float delta = p / (float)H + delta_bias;
  h1[(size_t)e * w + n] = act<T>::from_f(silu_f(wd1[n] * delta + bd1[n]));
}

template <typename T>
hipError_t launch_delta_hidden(const int64_t* t, const int64_t* t_obs, const int64_t* ages, int B, int H,
                               float delta_bias, const float* wd1, const float* bd1, int w, T* h1, hipStream_t s) {
  hipLaunchKernelGGL(delta_hidden_kernel<T>, dim3((w + 255) / 256, B), dim3(256), 0, s, t, t_obs, ages, B, H,
                     delta_bias, wd1, bd1, w, h1);
  return hipGetLastError();
}
template hipError_t launch_delta_hidden<float>(const int64_t*, const int64_t*, const int64_t*, int, int, float,
                                               const float*, const float*, int, float*, hipStream_t);
template hipError_t launch_delta_hidden<bf16_t>(const int64_t*, const int64_t*, const int64_t*, int, int, float,
                                                const float*, const float*, int, bf16_t*, hipStream_t);

// Offset of every env (concatenated to its slots' inputs): same age rule as the MLP's.
__global__ void offset_value_kernel(const int64_t* t, const int64_t* t_obs, const int64_t* ages, int B, int H,
                                    float delta_bias, double* dval) {
  const int e = blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= B) return;
  const double p = ages ? (double)ages[e] : (t ? (double)(*t - t_obs[e]) : 0.0);
  dval[e] = p / (double)H + (double)delta_bias;
}

hipError_t launch_offset_value(const int64_t* t, const int64_t* t_obs, const int64_t* ages, int B, int H,
                               float delta_bias, double* dval, hipStream_t s) {
  hipLaunchKernelGGL(offset_value_kernel, dim3((B + 255) / 256), dim3(256), 0, s, t, t_obs, ages, B, H, delta_bias,
                     dval);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Offset conditioning rows: cond[blk*H + i, n] = T(silu(ctau[i, n] + d[e, n]))
// ---------------------------------------------------------------------------
template <typename T>
__global__ void cond_expand_kernel(const float* __restrict__ d, int B, int H, int w, const float* __restrict__ ctau,
                                   int tau_row, const int* __restrict__ grp, T* __restrict__ cond) {
  // thread: 4 consecutive columns of one (env, slot) row
  const int i = blockIdx.y, e = blockIdx.z;
  const int ti = tau_row >= 0 ? tau_row : i;  // conditioning table row of this slot
  const int blk = grp ? grp[e] : e;
  if (blk < 0) return;
  const int n = (blockIdx.x * blockDim.x + threadIdx.x) * 4;
  if (n >= w) return;
  T* o = cond + ((size_t)blk * H + i) * w;
  if (n + 4 <= w && (w % 4) == 0) {
    const f32x4_t dv = d ? *(const f32x4_t*)(d + (size_t)e * w + n) : f32x4_t{0.f, 0.f, 0.f, 0.f};
    const f32x4_t c = *(const f32x4_t*)(ctau + (size_t)ti * w + n);
#pragma unroll
    for (int r = 0; r < 4; ++r) o[n + r] = act<T>::from_f(silu_f(c[r] + dv[r]));
    return;
  }
  for (int r = 0; r < 4 && n + r < w; ++r)
    o[n + r] = act<T>::from_f(silu_f(ctau[(size_t)ti * w + n + r] + (d ? d[(size_t)e * w + n + r] : 0.f)));
}

template <typename T>
hipError_t launch_cond_expand(const float* d, int B, int H, int w, const float* ctau, int tau_row, const int* grp,
                              T* cond, hipStream_t s) {
  hipLaunchKernelGGL(cond_expand_kernel<T>, dim3((w + 255) / 256, H, B), dim3(64), 0, s, d, B, H, w, ctau, tau_row,
                     grp, cond);
  return hipGetLastError();
}
template hipError_t launch_cond_expand<float>(const float*, int, int, int, const float*, int, const int*, float*,
                                              hipStream_t);
template hipError_t launch_cond_expand<bf16_t>(const float*, int, int, int, const float*, int, const int*, bf16_t*,
                                               hipStream_t);

// ---------------------------------------------------------------------------
// Offset conditioning of a few envs in one kernel: delta_e, h1 = silu(W_d1 delta +
// b_d1) (bf16, as the GEMM operand of the three-kernel path), d = W_d2 h1 + b_d2
// and cond[e*H + i, n] = bf16(silu(ctau[r, n] + d[n])).  Block = 4 waves over 16
// columns of one env; wave w owns columns 4w .. 4w+3 and its lanes split K in
// 8-element chunks (a wave reduction per column); h1 is formed by every block in
// LDS.  All of a block's loads are issued together at its start.
// ---------------------------------------------------------------------------
constexpr int kCondCols = 16;
constexpr int kCondMaxW = 2048;  // w <= 2048: 8 chunks of K per lane, 8 h1 values per thread
constexpr int kCondMaxH = 128;   // H <= 128: 8 conditioning entries per thread
// block (bx, by): columns [16 bx, 16 bx + 16) of env by
RAVEL_DEV void offset_cond_block(int bx, int by, const int64_t* t, const int64_t* t_obs, const int64_t* ages, int H,
                                 float delta_bias, const float* __restrict__ wd1, const float* __restrict__ bd1,
                                 const bf16_t* __restrict__ wd2, const float* __restrict__ bd2, int w,
                                 const float* __restrict__ ctau, int tau_row, bf16_t* __restrict__ cond) {
  __shared__ bf16_t h1[kCondMaxW];
  __shared__ float dcol[kCondCols];
  constexpr int MAXJ = kCondMaxW / 512, MAXK = kCondMaxW / 256, MAXC = kCondMaxH * kCondCols / 256;
  const int e = by, n0 = bx * kCondCols;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  // every load of the block is issued before any is used: the offset MLP's first
  // layer, this wave's four rows of W_d2, the conditioning table entries and bias
  float a1[MAXK], c1[MAXK];
#pragma unroll
  for (int q = 0; q < MAXK; ++q) {
    const int k = tid + 256 * q;
    a1[q] = k < w ? wd1[k] : 0.f;
    c1[q] = k < w ? bd1[k] : 0.f;
  }
  u32x4_t wv[4][MAXJ];
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    const int n = n0 + wave * 4 + c;
#pragma unroll
    for (int j = 0; j < MAXJ; ++j) {
      const int k = 8 * (lane + 64 * j);
      wv[c][j] = (n < w && k < w) ? *(const u32x4_t*)(wd2 + (size_t)n * w + k) : u32x4_t{0, 0, 0, 0};
    }
  }
  float cv[MAXC];
#pragma unroll
  for (int q = 0; q < MAXC; ++q) {
    const int idx = tid + 256 * q, i = idx / kCondCols, n = n0 + idx % kCondCols;
    const int ti = tau_row >= 0 ? tau_row : i;
    cv[q] = (i < H && n < w) ? ctau[(size_t)ti * w + n] : 0.f;
  }
  const float bias = (lane < 4 && n0 + wave * 4 + lane < w) ? bd2[n0 + wave * 4 + lane] : 0.f;
  const float p = ages ? (float)ages[e] : (t ? (float)(*t - t_obs[e]) : 0.f);
  const float delta = p / (float)H + delta_bias;
#pragma unroll
  for (int q = 0; q < MAXK; ++q) {
    const int k = tid + 256 * q;
    if (k < w) h1[k] = f32_to_bf16(silu_f(a1[q] * delta + c1[q]));
  }
  __syncthreads();
  // column n = n0 + 4 wave + c: lanes take 8-element chunks k = 8 (lane + 64 j)
  float acc[4];
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    float sacc = 0.f;
#pragma unroll
    for (int j = 0; j < MAXJ; ++j) {
      const int k = 8 * (lane + 64 * j);
      if (k >= w) break;
      const bf16_t* wb = reinterpret_cast<const bf16_t*>(&wv[c][j]);
#pragma unroll
      for (int q = 0; q < 8; ++q) sacc += bf16_to_f32(wb[q]) * bf16_to_f32(h1[k + q]);
    }
    acc[c] = wave_sum(sacc);
  }
  if (lane < 4) dcol[wave * 4 + lane] = (lane == 0 ? acc[0] : lane == 1 ? acc[1] : lane == 2 ? acc[2] : acc[3]) + bias;
  __syncthreads();
#pragma unroll
  for (int q = 0; q < MAXC; ++q) {
    const int idx = tid + 256 * q, i = idx / kCondCols, cc = idx % kCondCols, n = n0 + cc;
    if (i < H && n < w) cond[((size_t)e * H + i) * w + n] = f32_to_bf16(silu_f(cv[q] + dcol[cc]));
  }
}

__global__ __launch_bounds__(256) void offset_cond_kernel(const int64_t* t, const int64_t* t_obs,
                                                          const int64_t* ages, int H, float delta_bias,
                                                          const float* __restrict__ wd1,
                                                          const float* __restrict__ bd1,
                                                          const bf16_t* __restrict__ wd2,
                                                          const float* __restrict__ bd2, int w,
                                                          const float* __restrict__ ctau, int tau_row,
                                                          bf16_t* __restrict__ cond) {
  offset_cond_block(blockIdx.x, blockIdx.y, t, t_obs, ages, H, delta_bias, wd1, bd1, wd2, bd2, w, ctau, tau_row, cond);
}

hipError_t launch_offset_cond(const int64_t* t, const int64_t* t_obs, const int64_t* ages, int B, int H,
                              float delta_bias, const float* wd1, const float* bd1, const bf16_t* wd2,
                              const float* bd2, int w, const float* ctau, int tau_row, bf16_t* cond,
                              hipStream_t s) {
  if (w > kCondMaxW || w % 8 || B < 1 || H > kCondMaxH) return hipErrorInvalidValue;
  hipLaunchKernelGGL(offset_cond_kernel, dim3((w + kCondCols - 1) / kCondCols, B), dim3(256), 0, s, t, t_obs, ages, H,
                     delta_bias, wd1, bd1, wd2, bd2, w, ctau, tau_row, cond);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Input projection (logical slot order)
// ---------------------------------------------------------------------------
__global__ void transpose_f32_kernel(const float* __restrict__ src, int R, int C, float* __restrict__ dst) {
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= R * C) return;
  const int r = idx / C, c = idx % C;
  dst[(size_t)c * R + r] = src[idx];
}

hipError_t launch_transpose_f32(const float* src, int R, int C, float* dst, hipStream_t s) {
  hipLaunchKernelGGL(transpose_f32_kernel, dim3((R * C + 255) / 256), dim3(256), 0, s, src, R, C, dst);
  return hipGetLastError();
}

// Element (row, n) of a [w/32][64 rows][32] tile layout (rows < 64).
RAVEL_DEV size_t t32_index(int row, int n) { return ((size_t)(n >> 5) * 64 + row) * 32 + (n & 31); }

// bf16 copies of the norm shifts: item = 8 consecutive columns of one (chunk, row)
RAVEL_DEV void shift_copy_item(size_t idx, int M, int w, const InProjNorm& nrm) {
  const int per_row = w / 8;
  const size_t total = (size_t)nrm.cvt_chunks * M * per_row;
  if (idx >= total) return;
  const int n = (int)(idx % per_row) * 8;
  const int row = (int)((idx / per_row) % M);
  const int c = (int)(idx / ((size_t)per_row * M));
  const float* src = nrm.cvt_in + (size_t)row * nrm.cvt_ld + (size_t)c * nrm.cvt_stride + n;
  const f32x4_t a = *(const f32x4_t*)src, b = *(const f32x4_t*)(src + 4);
  const u32x4_t o = {pack_bf16x2(a[0], a[1]), pack_bf16x2(a[2], a[3]), pack_bf16x2(b[0], b[1]), pack_bf16x2(b[2], b[3])};
  *(u32x4_t*)(nrm.cvt_out + (size_t)c * 64 * w + t32_index(row, n)) = o;
}

// Block = 4 waves over 256 consecutive columns (one 64-column tile per wave) and
// rpb <= kInProjRows rows.  The weights are read transposed (w_inT[d, n]:
// consecutive lanes, consecutive addresses) once per block and kept in registers
// for all of its rows; the rows' ring entries are staged in LDS 16 features at a
// time, so a block costs one round of loads per 16 features whatever its row
// count.  Every output is bias + sum over d in increasing order.  Blocks past the
// row blocks (blockIdx.y >= nrowblk) make the bf16 shift copies instead.
constexpr int kInProjRows = 16;
// block (bx, by) of a (gx, ...) grid
RAVEL_DEV void in_proj_block(int bx, int by, int gx, const float* __restrict__ X, const int64_t* t, int B, int H, int D,
                             const float* __restrict__ w_inT, const float* __restrict__ b_in, int w,
                             float* __restrict__ x, const InProjNorm& nrm, const double* __restrict__ dval, int rpb,
                             int nrowblk) {
  __shared__ float xs[kInProjRows][16];
  const int tid = threadIdx.x;
  if (by >= nrowblk) {
    shift_copy_item(((size_t)(by - nrowblk) * gx + bx) * 256 + tid, B * H, w, nrm);
    return;
  }
  const int n = bx * 256 + tid;
  const int lane = tid & 63;
  const int BH = B * H;
  const int h0 = t ? (int)(*t % H) : 0;  // no step counter: X is a chunk in logical order
  const int row0 = by * rpb;
  const int nrows = min(rpb, BH - row0);
  // the first norm's scales of this thread's column, requested up front
  float scv[kInProjRows];
#pragma unroll
  for (int rr = 0; rr < kInProjRows; ++rr)
    scv[rr] = (nrm.p && rr < nrows && n < w) ? nrm.scale[(size_t)(row0 + rr) * nrm.ldm + n] : 0.f;
  // thread (sr, sj) stages feature d0 + sj of row row0 + sr
  const int sr = tid >> 4, sj = tid & 15;
  const float* srow = nullptr;
  if (sr < nrows) {
    const int row = row0 + sr, e = row / H, i = row % H;
    const int ph = h0 + i < H ? h0 + i : h0 + i - H;
    srow = X + ((size_t)e * H + ph) * D;
  }
  float acc[kInProjRows];
  const float bias = n < w ? b_in[n] : 0.f;
#pragma unroll
  for (int rr = 0; rr < kInProjRows; ++rr) acc[rr] = bias;
  for (int d0 = 0; d0 < D; d0 += 16) {
    float wv[16];
#pragma unroll
    for (int j = 0; j < 16; ++j) wv[j] = (n < w && d0 + j < D) ? w_inT[(size_t)(d0 + j) * w + n] : 0.f;
    const float xv = (srow && d0 + sj < D) ? srow[d0 + sj] : 0.f;
    __syncthreads();  // the previous chunk's reads are done
    xs[sr][sj] = xv;
    __syncthreads();
#pragma unroll
    for (int rr = 0; rr < kInProjRows; ++rr)
      if (rr < nrows) {
#pragma unroll
        for (int j = 0; j < 16; ++j) acc[rr] += wv[j] * xs[rr][j];
      }
  }
  if (dval) {  // the offset as input feature D of every slot
    const float wd = n < w ? w_inT[(size_t)D * w + n] : 0.f;
#pragma unroll
    for (int rr = 0; rr < kInProjRows; ++rr)
      if (rr < nrows) acc[rr] += wd * (float)dval[(row0 + rr) / H];
  }
#pragma unroll
  for (int rr = 0; rr < kInProjRows; ++rr) {
    if (rr >= nrows) break;
    const int row = row0 + rr;
    if (n < w) x[(size_t)row * w + n] = acc[rr];
    if (!nrm.sumsq) continue;
    // first adaptive norm of the persistent step: p = bf16((1 + scale) x) (unless the
    // modulation GEMM forms it), the 64-column tile's sum of squares of the row, and
    // the bf16 shift copies
    const float v = n < w ? acc[rr] : 0.f;
    if (nrm.p && n < w) nrm.p[t32_index(row, n)] = f32_to_bf16((1.f + scv[rr]) * v);
    const float sq = wave_sum(v * v);
    if (lane == 0 && n < w) nrm.sumsq[(size_t)(n >> 6) * 64 + row] = sq;
  }
}

__global__ __launch_bounds__(256) void in_proj_kernel(const float* __restrict__ X, const int64_t* t, int B, int H, int D,
                                                      const float* __restrict__ w_inT, const float* __restrict__ b_in,
                                                      int w, float* __restrict__ x, InProjNorm nrm,
                                                      const double* __restrict__ dval, int rpb, int nrowblk) {
  in_proj_block(blockIdx.x, blockIdx.y, gridDim.x, X, t, B, H, D, w_inT, b_in, w, x, nrm, dval, rpb, nrowblk);
}

// The offset conditioning (blocks [0, ncx * B)) and the input projection with the
// rows' sums of squares (the rest, one row per block) of a few-row step in one
// launch: neither reads the other's output.
__global__ __launch_bounds__(256) void offset_cond_in_proj_kernel(
    const int64_t* t, const int64_t* t_obs, int H, float delta_bias, const float* __restrict__ wd1,
    const float* __restrict__ bd1, const bf16_t* __restrict__ wd2, const float* __restrict__ bd2, int w,
    const float* __restrict__ ctau, bf16_t* __restrict__ cond, int ncx, int nc, const float* __restrict__ X, int B,
    int D, const float* __restrict__ w_inT, const float* __restrict__ b_in, float* __restrict__ x, InProjNorm nrm,
    int ipx, int nrowblk) {
  const int b = blockIdx.x;
  if (b < nc) {
    offset_cond_block(b % ncx, b / ncx, t, t_obs, nullptr, H, delta_bias, wd1, bd1, wd2, bd2, w, ctau, -1, cond);
  } else {
    const int i = b - nc;
    in_proj_block(i % ipx, i / ipx, ipx, X, t, B, H, D, w_inT, b_in, w, x, nrm, nullptr, 1, nrowblk);
  }
}

hipError_t launch_offset_cond_in_proj(const int64_t* t, const int64_t* t_obs, int B, int H, float delta_bias,
                                      const float* wd1, const float* bd1, const bf16_t* wd2, const float* bd2, int w,
                                      const float* ctau, bf16_t* cond, const float* X, int D, const float* w_inT,
                                      const float* b_in, float* x, float* sumsq, hipStream_t s) {
  if (w > kCondMaxW || w % 64 || B < 1 || H > kCondMaxH || B * H > 64 || !t || !sumsq) return hipErrorInvalidValue;
  InProjNorm nrm{};
  nrm.sumsq = sumsq;
  const int ncx = (w + kCondCols - 1) / kCondCols, nc = ncx * B;
  const int ipx = (w + 255) / 256, nrowblk = B * H;
  hipLaunchKernelGGL(offset_cond_in_proj_kernel, dim3(nc + ipx * nrowblk), dim3(256), 0, s, t, t_obs, H, delta_bias,
                     wd1, bd1, wd2, bd2, w, ctau, cond, ncx, nc, X, B, D, w_inT, b_in, x, nrm, ipx, nrowblk);
  return hipGetLastError();
}

hipError_t launch_in_proj(const float* X, const int64_t* t, int B, int H, int D, const float* w_inT,
                          const float* b_in, int w, float* x, const InProjNorm& nrm, const double* dval,
                          hipStream_t s) {
  if (nrm.p && (B * H > 64 || (w % 64) != 0)) return hipErrorInvalidValue;
  // many rows: 16 per block; few rows: one per block (more blocks, same chain per block)
  const int BH = B * H;
  const int rpb = BH >= 1024 ? kInProjRows : (BH >= 256 ? 4 : 1);
  const int cols = (w + 255) / 256, nrowblk = (BH + rpb - 1) / rpb;
  // the shift copies ride along in extra row blocks of the same launch
  int extra = 0;
  if (nrm.p && nrm.cvt_chunks > 0) {
    const size_t total = (size_t)nrm.cvt_chunks * BH * (w / 8);
    extra = (int)((total + (size_t)cols * 256 - 1) / ((size_t)cols * 256));
  }
  hipLaunchKernelGGL(in_proj_kernel, dim3(cols, nrowblk + extra), dim3(256), 0, s, X, t, B, H, D, w_inT, b_in, w, x, nrm,
                     dval, rpb, nrowblk);
  return hipGetLastError();
}

// Block = 4 waves over 256 consecutive columns of one row (blockIdx.y < BH), or
// shift copies (blockIdx.y >= BH): the in_proj_kernel epilogue for rows that
// were produced elsewhere.
__global__ __launch_bounds__(256) void norm_operands_kernel(const float* __restrict__ x, int BH, int w,
                                                            InProjNorm nrm) {
  const int tid = threadIdx.x;
  if ((int)blockIdx.y >= BH) {
    shift_copy_item(((size_t)(blockIdx.y - BH) * gridDim.x + blockIdx.x) * 256 + tid, BH, w, nrm);
    return;
  }
  const int row = blockIdx.y, n = blockIdx.x * 256 + tid;
  // w is a multiple of 64: a wave is wholly inside or wholly outside the row
  if (n >= w) return;
  const float v = x[(size_t)row * w + n];
  nrm.p[t32_index(row, n)] = f32_to_bf16((1.f + nrm.scale[(size_t)row * nrm.ldm + n]) * v);
  const float sq = wave_sum(v * v);
  if ((tid & 63) == 0) nrm.sumsq[(size_t)(n >> 6) * 64 + row] = sq;
}

hipError_t launch_norm_operands(const float* x, int BH, int w, const InProjNorm& nrm, hipStream_t s) {
  if (!nrm.p || BH <= 0 || BH > 64 || (w % 64) != 0) return hipErrorInvalidValue;
  const int cols = (w + 255) / 256;
  int extra = 0;
  if (nrm.cvt_chunks > 0) {
    const size_t total = (size_t)nrm.cvt_chunks * BH * (w / 8);
    extra = (int)((total + (size_t)cols * 256 - 1) / ((size_t)cols * 256));
  }
  hipLaunchKernelGGL(norm_operands_kernel, dim3(cols, BH + extra), dim3(256), 0, s, x, BH, w, nrm);
  return hipGetLastError();
}

// Sinusoid of value v at column c of a w-wide embedding (c < w/2: sine, else
// cosine), as the flow-time embedding, in float64.
RAVEL_DEV float sinusoid_at(double v, int c, int w) {
  const int half = w / 2;
  const int jj = c < half ? c : c - half;
  const double arg = 1000.0 * v * pow(10000.0, -(double)jj / (double)half);
  return (float)(c < half ? sin(arg) : cos(arg));
}

// One block column range of one row; grid (ceil(ldz / 256), B * H).
template <typename T>
__global__ __launch_bounds__(256) void offset_rows_kernel(int mode, const float* __restrict__ x,
                                                          const double* __restrict__ dval, int H, int w, int tau_row,
                                                          int tau_den, T* __restrict__ z, int ldz) {
  const int row = blockIdx.y, e = row / H, i = row % H;
  const double dv = dval[e];
  // mode 0: the slot's flow time; mode 1: the env's offset
  const double tv = mode == 1 ? dv : (tau_row < 0 ? (double)(i + 1) / (double)H
                                                  : (double)(tau_row + 1) / (double)tau_den);
  const float* xr = x + (size_t)row * w;
  T* zr = z + (size_t)row * ldz;
  for (int c = blockIdx.x * 256 + threadIdx.x; c < ldz; c += gridDim.x * 256) {
    float v = 0.f;
    if (c < w)
      v = xr[c];
    else if (c < 2 * w)
      v = sinusoid_at(tv, c - w, w);
    else if (mode == 0 && c == 2 * w)
      v = (float)dv;
    zr[c] = act<T>::from_f(v);
  }
}

template <typename T>
hipError_t launch_offset_rows(int mode, const float* x, const double* dval, int B, int H, int w, int tau_row,
                              int tau_den, T* z, int ldz, hipStream_t s) {
  if (B <= 0 || (w % 2) || ldz < 2 * w + (mode == 0 ? 1 : 0) || (tau_row >= 0 && tau_den <= 0))
    return hipErrorInvalidValue;
  hipLaunchKernelGGL(offset_rows_kernel<T>, dim3((ldz + 255) / 256, B * H), dim3(256), 0, s, mode, x, dval, H, w,
                     tau_row, tau_den, z, ldz);
  return hipGetLastError();
}
template hipError_t launch_offset_rows<float>(int, const float*, const double*, int, int, int, int, int, float*, int,
                                              hipStream_t);
template hipError_t launch_offset_rows<bf16_t>(int, const float*, const double*, int, int, int, int, int, bf16_t*,
                                               int, hipStream_t);

// Rotary position embedding in place; grid (ceil(nh * hd/2 / 256), B * H), one thread per pair.
template <typename T>
__global__ __launch_bounds__(256) void rope_kernel(T* __restrict__ qkv, int ld, int H, int nh, int hd,
                                                   const float* __restrict__ cs) {
  const int row = blockIdx.y, i = row % H, half = hd / 2;
  const int idx = blockIdx.x * 256 + threadIdx.x;
  if (idx >= nh * half) return;
  const int h = idx / half, d = idx - h * half;
  T* p = qkv + (size_t)row * ld + (size_t)h * hd + d;
  const float c = cs[((size_t)i * half + d) * 2], sn = cs[((size_t)i * half + d) * 2 + 1];
  const float a = act<T>::to_f(p[0]), b = act<T>::to_f(p[half]);
  p[0] = act<T>::from_f(a * c - b * sn);
  p[half] = act<T>::from_f(b * c + a * sn);
}

template <typename T>
hipError_t launch_rope(T* qkv, int ld, int BH, int H, int nq, int nkv, int hd, const float* cs, hipStream_t s) {
  const int nh = nq + nkv;
  if (BH <= 0 || H <= 0 || BH % H || (hd % 2) || ld < nh * hd) return hipErrorInvalidValue;
  hipLaunchKernelGGL(rope_kernel<T>, dim3((nh * (hd / 2) + 255) / 256, BH), dim3(256), 0, s, qkv, ld, H, nh, hd, cs);
  return hipGetLastError();
}
template hipError_t launch_rope<float>(float*, int, int, int, int, int, int, const float*, hipStream_t);
template hipError_t launch_rope<bf16_t>(bf16_t*, int, int, int, int, int, int, const float*, hipStream_t);

// ---------------------------------------------------------------------------
// Analytic velocity fields
// ---------------------------------------------------------------------------
__global__ void analytic_velocity_kernel(int kind, const float* __restrict__ X, const int64_t* t, int B,
                                         int H, int D, const float* __restrict__ param, float tau_all,
                                         const float* __restrict__ state, const float* __restrict__ mask,
                                         float* __restrict__ v) {
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= B * H * D) return;
  const int d = idx % D, i = (idx / D) % H, e = idx / (D * H);
  const int ph = t ? (int)((*t + i) % H) : i;
  const float x = X[((size_t)e * H + ph) * D + d];
  float out;
  if (kind == 1) {  // OT: (x - a*) / tau, tau_i = (i+1)/H on the ring, tau_all for a chunk
    const float tau = tau_all > 0.f ? tau_all : (float)(i + 1) / (float)H;
    // an absolute target is aimed at relative to the state on relative dimensions
    const float target = state ? param[d] - mask[d] * state[(size_t)e * D + d] : param[d];
    out = (x - target) / tau;
  } else {  // LINEAR: lambda * x
    out = param[0] * x;
  }
  v[idx] = out;
}

hipError_t launch_analytic_velocity(int kind, const float* X, const int64_t* t, int B, int H, int D,
                                    const float* param, float tau_all, const float* state, const float* mask,
                                    float* v, hipStream_t s) {
  const int n = B * H * D;
  hipLaunchKernelGGL(analytic_velocity_kernel, dim3((n + 255) / 256), dim3(256), 0, s, kind, X, t, B, H, D,
                     param, tau_all, state, mask, v);
  return hipGetLastError();
}

// Relative actions: re-express every slot's clean part against the new state,
// X[e, (t+i) mod H, d] += (1 - tau_i) * mask[d] * (s_prev[e, d] - state[e, d]) (no shift at an
// env's first step), then s_prev = state.  One block per env.
__global__ __launch_bounds__(256) void relative_shift_kernel(float* __restrict__ X, const int64_t* t, int H, int D,
                                                             const float* __restrict__ mask,
                                                             const float* __restrict__ state,
                                                             float* __restrict__ s_prev, int* __restrict__ has_prev) {
#pragma clang fp contract(off)
  const int e = blockIdx.x;
  const int h0 = (int)(*t % H);
  const float* st = state + (size_t)e * D;
  float* sp = s_prev + (size_t)e * D;
  if (has_prev[e]) {
    for (int k = threadIdx.x; k < H * D; k += blockDim.x) {
      const int i = k / D, d = k % D;
      int ph = h0 + i;
      if (ph >= H) ph -= H;
      const float tau = (float)(i + 1) / (float)H;
      const float shift = mask[d] * (sp[d] - st[d]);
      const float step = (1.0f - tau) * shift;
      float* xp = X + ((size_t)e * H + ph) * D + d;
      *xp = *xp + step;
    }
  }
  __syncthreads();
  for (int d = threadIdx.x; d < D; d += blockDim.x) sp[d] = st[d];
  if (threadIdx.x == 0) has_prev[e] = 1;
}

hipError_t launch_relative_shift(float* X, const int64_t* t, int B, int H, int D, const float* mask,
                                 const float* state, float* s_prev, int* has_prev, hipStream_t s) {
  hipLaunchKernelGGL(relative_shift_kernel, dim3(B), dim3(256), 0, s, X, t, H, D, mask, state, s_prev, has_prev);
  return hipGetLastError();
}


// ---------------------------------------------------------------------------
// Euler update + release + noise append + step counter
// ---------------------------------------------------------------------------
// x <- x - dt * v with a separately rounded product (no fused multiply-add), the
// exact operation order of the reference definition.
RAVEL_DEV float euler_sub(float x, float dt, float v) {
#pragma clang fp contract(off)
  const float step = dt * v;
  return x - step;
}

// Euler step of a full-horizon chunk: X[e, i, :] -= dt * v[e*H + i, :] for every slot.
__global__ void euler_chunk_kernel(float* __restrict__ X, const float* __restrict__ v, int n, float dt) {
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;
  if (idx < n) X[idx] = euler_sub(X[idx], dt, v[idx]);
}

hipError_t launch_euler_chunk(float* X, const float* v, int B, int H, int D, float dt, hipStream_t s) {
  const int n = B * H * D;
  hipLaunchKernelGGL(euler_chunk_kernel, dim3((n + 255) / 256), dim3(256), 0, s, X, v, n, dt);
  return hipGetLastError();
}

// Training buffer at the rolling flow-time profile: X[e, i, :] = tau_i * noise + (1 - tau_i) * target,
// tau_i = (i+1)/H, each product rounded on its own (the definition's operation order).
__global__ void train_buffer_kernel(const float* __restrict__ target, const float* __restrict__ noise, int B, int H,
                                    int D, float* __restrict__ X) {
#pragma clang fp contract(off)
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= B * H * D) return;
  const int i = (idx / D) % H;
  const float tau = (float)(i + 1) / (float)H;
  const float a = tau * noise[idx];
  const float c = (1.0f - tau) * target[idx];
  X[idx] = a + c;
}

hipError_t launch_train_buffer(const float* target, const float* noise, int B, int H, int D, float* X, hipStream_t s) {
  const int n = B * H * D;
  hipLaunchKernelGGL(train_buffer_kernel, dim3((n + 255) / 256), dim3(256), 0, s, target, noise, B, H, D, X);
  return hipGetLastError();
}

// Flow-matching loss per sample: loss[e] = (1/H) sum_i ||v[e*H+i] - (noise - target)[e, i]||^2.
// One block per sample, a fixed reduction order (deterministic).
__global__ __launch_bounds__(256) void train_loss_kernel(const float* __restrict__ v, const float* __restrict__ target,
                                                         const float* __restrict__ noise, int H, int D,
                                                         float* __restrict__ loss) {
  __shared__ float part[4];
  const int e = blockIdx.x, tid = threadIdx.x;
  const size_t base = (size_t)e * H * D;
  float acc = 0.f;
  for (int k = tid; k < H * D; k += 256) {
    const float r = v[base + k] - (noise[base + k] - target[base + k]);
    acc += r * r;
  }
  acc = wave_sum(acc);
  if ((tid & 63) == 0) part[tid >> 6] = acc;
  __syncthreads();
  if (tid == 0) loss[e] = ((part[0] + part[1]) + (part[2] + part[3])) / (float)H;
}

hipError_t launch_train_loss(const float* v, const float* target, const float* noise, int B, int H, int D, float* loss,
                             hipStream_t s) {
  hipLaunchKernelGGL(train_loss_kernel, dim3(B), dim3(256), 0, s, v, target, noise, H, D, loss);
  return hipGetLastError();
}

// One block per env: each thread applies the Euler update to its ring elements and,
// for logical slot 0, releases the updated value as the action and refills the
// slot with the noise of the new tail step.  Every block reads the step counter at
// its start; a single block advances it once its threads have read it, several
// blocks take a ticket and the last one advances it (and re-arms the ticket).
__global__ __launch_bounds__(256) void euler_release_kernel(float* __restrict__ X, const float* __restrict__ v,
                                                            int64_t* t, int H, int D, uint64_t seed,
                                                            float* __restrict__ action,
                                                            const float* __restrict__ state,
                                                            const float* __restrict__ mask, unsigned* ticket,
                                                            const int* err, int* host_flag) {
  // The layers' kernel reported a failure (a grid barrier that timed out): v is not
  // a velocity.  Release NaN actions, leave the ring and t as they were, and raise
  // the host-visible flag that the next step call checks.
  if (err && __hip_atomic_load(err, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0) {
    for (int d = threadIdx.x; d < D; d += blockDim.x) action[(size_t)blockIdx.x * D + d] = __int_as_float(0x7fc00000);
    if (host_flag && blockIdx.x == 0 && threadIdx.x == 0)
      __hip_atomic_store(host_flag, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
    return;
  }
  const int64_t tt = *t;
  const float dt = 1.0f / (float)H;
  const int h0 = (int)(tt % H);
  const int e = blockIdx.x;
  const int n = H * D;
  float* Xe = X + (size_t)e * H * D;
  const float* ve = v + (size_t)e * H * D;
  // logical slot i of element k = i * D + d sits in physical slot (h0 + i) mod H;
  // 4 elements per thread per batch, loads first
  for (int k0 = 0; k0 < n; k0 += 4 * 256) {
    float xv[4], vv[4];
    int off[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int k = k0 + u * 256 + (int)threadIdx.x;
      const int i = k / D, d = k - i * D;
      int ph = h0 + i;
      if (ph >= H) ph -= H;
      off[u] = k < n ? ph * D + d : -1;
      xv[u] = k < n ? Xe[off[u]] : 0.f;
      vv[u] = k < n ? ve[k] : 0.f;
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      if (off[u] < 0) continue;
      const float xn = euler_sub(xv[u], dt, vv[u]);
      const int k = k0 + u * 256 + (int)threadIdx.x;
      if (k >= D) {
        Xe[off[u]] = xn;
        continue;
      }
      // logical slot 0 (k = d): released; its slot becomes the tail, refilled with the
      // noise of step tt + H (4 dimensions per noise draw)
      const int d = k;
      action[(size_t)e * D + d] = state ? xn + mask[d] * state[(size_t)e * D + d] : xn;
      float z[4];
      ring_noise4(seed, e, tt + H, d >> 2, z);
      Xe[off[u]] = z[d & 3];
    }
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    if (gridDim.x == 1) {
      *t = tt + 1;
    } else {
      const unsigned prev = atomicAdd(ticket, 1u);
      if (prev == gridDim.x - 1) {
        *ticket = 0u;
        *t = tt + 1;
      }
    }
  }
}

hipError_t launch_euler_release(float* X, const float* v, int64_t* t, int B, int H, int D, uint64_t seed,
                                float* action, unsigned* ticket, const float* state, const float* mask,
                                const int* err, int* host_flag, hipStream_t s) {
  if (!ticket) return hipErrorInvalidValue;
  hipLaunchKernelGGL(euler_release_kernel, dim3(B), dim3(256), 0, s, X, v, t, H, D, seed, action, state, mask,
                     ticket, err, host_flag);
  return hipGetLastError();
}

__global__ void zero_u32_kernel(unsigned* __restrict__ p, long long n) {
  const long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = 0u;
}

// Zero n words with a kernel (a memset node recorded into a captured graph is avoided).
hipError_t launch_zero_u32(unsigned* p, long long n, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(zero_u32_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, p, n);
  return hipGetLastError();
}

__global__ void ring_init_kernel(float* X, int B, int H, int D, uint64_t seed) {
  const int NG = (D + 3) / 4;
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= B * H * NG) return;
  const int c = idx % NG, r = (idx / NG) % H, e = idx / (NG * H);
  float z[4];
  ring_noise4(seed, e, r, c, z);
  for (int q = 0; q < 4; ++q) {
    const int d = c * 4 + q;
    if (d < D) X[((size_t)e * H + (r % H)) * D + d] = z[q];
  }
}

hipError_t launch_ring_init(float* X, int B, int H, int D, uint64_t seed, hipStream_t s) {
  const int n = B * H * ((D + 3) / 4);
  hipLaunchKernelGGL(ring_init_kernel, dim3((n + 255) / 256), dim3(256), 0, s, X, B, H, D, seed);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Flow-time embedding (float64)
// ---------------------------------------------------------------------------
template <typename T>
__global__ void time_embedding_kernel(int H, int w, T* emb) {
  const int half = w / 2;
  const int idx = blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= H * half) return;
  const int i = idx / half, jj = idx % half;
  const double tau = (double)(i + 1) / (double)H;
  const double omega = pow(10000.0, -(double)jj / (double)half);
  const double arg = 1000.0 * tau * omega;
  emb[(size_t)i * w + jj] = act<T>::from_f((float)sin(arg));
  emb[(size_t)i * w + half + jj] = act<T>::from_f((float)cos(arg));
}

template <typename T>
hipError_t launch_time_embedding(int H, int w, T* emb, hipStream_t s) {
  const int n = H * (w / 2);
  hipLaunchKernelGGL(time_embedding_kernel<T>, dim3((n + 255) / 256), dim3(256), 0, s, H, w, emb);
  return hipGetLastError();
}
template hipError_t launch_time_embedding<float>(int, int, float*, hipStream_t);
template hipError_t launch_time_embedding<bf16_t>(int, int, bf16_t*, hipStream_t);

// ---------------------------------------------------------------------------
// Utilities
// ---------------------------------------------------------------------------
template <typename T>
__global__ void convert_kernel(const float* __restrict__ src, T* __restrict__ dst, long long n) {
  const long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) dst[i] = act<T>::from_f(src[i]);
}

template <typename T>
hipError_t launch_convert(const float* src, T* dst, long long n, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(convert_kernel<T>, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, src, dst, n);
  return hipGetLastError();
}
template hipError_t launch_convert<float>(const float*, float*, long long, hipStream_t);
template hipError_t launch_convert<bf16_t>(const float*, bf16_t*, long long, hipStream_t);

__global__ void publish_kernel(PublishBatch pb, int* slot, int64_t* t_obs) {
  const int i = threadIdx.x;
  if (i < pb.n) {
    slot[pb.env[i]] = pb.new_slot[i];
    t_obs[pb.env[i]] = pb.tobs[i];
  }
}

hipError_t launch_publish(const PublishBatch& pb, int* slot, int64_t* t_obs, hipStream_t s) {
  hipLaunchKernelGGL(publish_kernel, dim3(1), dim3(32), 0, s, pb, slot, t_obs);
  return hipGetLastError();
}

template <typename T>
__global__ void check_finite_kernel(const T* p, long long n, int* flag) {
  const long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) {
    const float v = act<T>::to_f(p[i]);
    if (!isfinite(v)) atomicOr(flag, 1);
  }
}

hipError_t launch_check_finite(const float* p, long long n, int* flag, hipStream_t s) {
  return launch_check_finite_t<float>(p, n, flag, s);
}

template <typename T>
hipError_t launch_check_finite_t(const T* p, long long n, int* flag, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  hipLaunchKernelGGL(check_finite_kernel<T>, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, s, p, n, flag);
  return hipGetLastError();
}
template hipError_t launch_check_finite_t<float>(const float*, long long, int*, hipStream_t);
template hipError_t launch_check_finite_t<bf16_t>(const bf16_t*, long long, int*, hipStream_t);

}  // namespace ravel
