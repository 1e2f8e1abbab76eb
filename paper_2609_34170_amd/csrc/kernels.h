// Kernel launch interface of libravel (internal; not part of the C ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "common.h"

namespace ravel {

// Device-scope tickets (split-K tiles, attention key splits) are spaced one per
// 256 bytes so that atomics of different tiles never share a cache line.
#ifndef RAVEL_COUNTER_STRIDE
#define RAVEL_COUNTER_STRIDE 64
#endif
constexpr int kCounterStride = RAVEL_COUNTER_STRIDE;

// ---------------------------------------------------------------------------
// GEMM  C[M,N] = A[M,K] . B[N,K]^T  (both operands K-contiguous), fp32 accumulate,
// followed by a fused epilogue.
// ---------------------------------------------------------------------------
enum EpiMode {
  EPI_F32 = 0,        // out_f[m,n]  = acc + bias[n]
  EPI_T = 1,          // out_t[m,n]  = T(acc + bias[n])
  EPI_RESID = 2,      // out_f[m,n] += gate[m,n] * acc            (gated residual)
  EPI_RESID_TANH = 3, // out_f[m,n] += tanh(*gate_scalar) * acc    (adapter gate)
  EPI_GEGLU = 4,      // out_t[m,f]  = T(gelu_tanh(acc_gate) * acc_up), columns interleaved
                      //               in blocks of 16 gate / 16 up (N = 2F)
  EPI_COND = 5,       // out_t[m*H+i, n] = T(silu(ctau[i,n] + acc + bias[n])) for i < H
  EPI_GELU_T = 6,     // out_t[m,n]  = T(gelu_tanh(acc + bias[n]))
  EPI_SILU_T = 7,     // out_t[m,n]  = T(silu(acc + bias[n]))
};

struct GemmArgs {
  const void* A; int lda;
  const void* B; int ldb;
  int M, N, K;
  int ksplit;          // number of K ranges (grid.z); 1 = no split
  int kchunk;          // K elements per range (multiple of 64)
  float* partial;      // split-K workspace: ksplit x tiles x tile elements, fp32
  unsigned* counters;  // one per output tile, zero; the reducing block re-zeroes it
  int mode;
  const float* bias;
  float* out_f; int ldo_f;
  void* out_t; int ldo_t;
  const float* gate; int ldg;
  const float* gate_scalar;
  const float* ctau; int H;
  // Rows that share their modulation (see launch_cond_groups); all optional:
  const int* m_rows;     // device row count: rows >= min(M, *m_rows) are neither computed nor stored
  const int* gate_rows;  // [M]: EPI_RESID reads gate row gate_rows[m] instead of row m
  const int* cond_grp;   // [M], EPI_COND: output block cond_grp[m] (>= 0), or nothing (< 0)
  // Whole-K few-row kernel, EPI_F32 on a layer's modulation rows (value v = acc + bias
  // at columns [0, 6 nrm_w)): also the first adaptive norm's operands, p[m][n] =
  // bf16((1 + v[m][n]) nrm_x[m][n]) for n < nrm_w, and bf16 copies of the two shifts
  // (columns [nrm_w, 2 nrm_w) and [4 nrm_w, 5 nrm_w)) as chunks 0 and 1 of nrm_shift;
  // p and the chunks (64 * nrm_w elements apart) in 32-column tiles [nrm_w/32][64][32].
  bf16_t* nrm_p;
  const float* nrm_x;
  bf16_t* nrm_shift;
  int nrm_w;
};

// Tile configurations of the bf16 MFMA GEMM.
enum GemmTile {
  TILE_64x64 = 0, TILE_128x128 = 1, TILE_64x128 = 2, TILE_128x64 = 3, TILE_32x64 = 4,
  TILE_256x128 = 5, TILE_128x256 = 6, TILE_256x256 = 7
};

hipError_t launch_gemm_bf16(const GemmArgs& a, int tile, hipStream_t s);
// M <= 64 weight-streaming kernel: block columns 64*nfr (nfr 1 or 2, 2 for EPI_GEGLU),
// K range per block kchunk in {128, 256, 512} (1024 with nfr 1), ksplit ranges (grid.y).
hipError_t launch_gemm_skinny(const GemmArgs& a, int nfr, hipStream_t s);
// M <= 64, 64-column tiles, waves split the block's K range (kchunk 256 or 512 = 4 or 8
// waves), ksplit ranges (grid.y).
hipError_t launch_gemm_regstream(const GemmArgs& a, hipStream_t s);
// M <= 64, K <= 1024 with K % 128 == 0, not EPI_GEGLU: 32-column blocks over the whole
// K, waves split it in quarters (no split-K workspace).
hipError_t launch_gemm_wholek(const GemmArgs& a, hipStream_t s);
// Two whole-K few-row GEMMs in one launch (blocks of a1 first, then those of a2).
hipError_t launch_gemm_wholek2(const GemmArgs& a1, const GemmArgs& a2, hipStream_t s);
hipError_t launch_gemm_f32(const GemmArgs& a, hipStream_t s);

// ---------------------------------------------------------------------------
// Attention: per env e and query head j, softmax(q K^T * scale) V over the keys
// [prefix tokens of env e ; S self tokens of env e], no mask, GQA head map
// g = j * nkv / nq.
// ---------------------------------------------------------------------------
struct AttnArgs {
  const void* q; int ldq;          // q[(e*Hq + i)*ldq + j*hd + d]
  int Hq;                          // queries per env
  const void* pk; const void* pv;  // prefix rows: base + slot*slot_stride + e*env_stride + p*p_ld + g*hd
  long long p_env_stride, p_slot_stride;
  const int* slot;                 // [B] active context slot or null
  int P, p_ld;
  const void* sk; const void* sv;  // self rows: base + (e*S + s)*s_ld + g*hd
  int S, s_ld;
  int B, nq, nkv, hd;
  float scale;
  void* out; int ldo;              // out[(e*Hq + i)*ldo + j*hd + d]
  int nsplit, keys_per_split;      // split of the key range (multiple of 32)
  float* part_o;                   // [B*nq*nsplit][Hq_pad][hd] (persistent kernel: fp16, normalised)
  float* part_ml;                  // [B*nq*nsplit][Hq_pad][2]
  unsigned* counters;              // [B*nq]
  int coop;                        // persistent kernel: the splits of a head merge together
  int coh;                         // persistent kernel: device-coherent loads of q and the self rows
};

hipError_t launch_attn_bf16(const AttnArgs& a, hipStream_t s);
hipError_t launch_attn_f32(const AttnArgs& a, hipStream_t s);

// ---------------------------------------------------------------------------
// Element-wise / row kernels
// ---------------------------------------------------------------------------
// y[m,:] = T( x/rms(x) * (1 + scale) + shift ), per-row modulation rows of stride ldm
// (mode 0) or a per-feature scale without shift (mode 1: scale[n], shift ignored).
// With rowmap (mode 0), row m takes its scale/shift from row rowmap[m].
template <typename T>
hipError_t launch_adarms(const float* x, int ldx, int M, int w, const float* scale,
                         const float* shift, int ldm, int mode, const int* rowmap, float eps, T* y, int ldy,
                         hipStream_t s);
// Groups of envs whose offset conditioning is identical within a step (equal
// observation time t_obs, hence equal context age and delta): group g is the
// g-th distinct t_obs in env order.  grp[e] = g for the first env of its group
// and -1 - g for the others; rowmap[e*H + i] = g*H + i; *rows = (#groups)*H.
// One block; B <= kCondGroupsMaxB.
constexpr int kCondGroupsMaxB = 1024;
hipError_t launch_cond_groups(const int64_t* t_obs, int B, int H, int* grp, int* rowmap, int* rows,
                              hipStream_t s);

// Offset conditioning hidden layer: h1[e,n] = T(silu(wd1[n]*delta_e + bd1[n])),
// delta_e = p_e / H + delta_bias with context age p_e = ages[e] if ages is given, else
// t - t_obs[e], or 0 when t is NULL too.
template <typename T>
hipError_t launch_delta_hidden(const int64_t* t, const int64_t* t_obs, const int64_t* ages, int B, int H,
                               float delta_bias, const float* wd1, const float* bd1, int w, T* h1, hipStream_t s);

// Training buffer at the rolling profile: X[e,i,:] = tau_i noise + (1 - tau_i) target, tau_i = (i+1)/H.
hipError_t launch_train_buffer(const float* target, const float* noise, int B, int H, int D, float* X, hipStream_t s);
// Flow-matching loss per sample: loss[e] = (1/H) sum_i ||v[e*H+i,:] - (noise - target)[e,i,:]||^2.
hipError_t launch_train_loss(const float* v, const float* target, const float* noise, int B, int H, int D, float* loss,
                             hipStream_t s);

// Offset conditioning rows: cond[blk*H + i, n] = T(silu(ctau[r, n] + d[e, n])) for every env e
// with blk = grp[e] (>= 0; envs with grp[e] < 0 write nothing) or blk = e without grp, and
// table row r = i (tau_row < 0: each slot its own flow time) or r = tau_row (every slot);
// d = NULL: no offset term.
template <typename T>
hipError_t launch_cond_expand(const float* d, int B, int H, int w, const float* ctau, int tau_row, const int* grp,
                              T* cond, hipStream_t s);

// dst[c, r] = src[r, c] for an R x C fp32 matrix.
hipError_t launch_transpose_f32(const float* src, int R, int C, float* dst, hipStream_t s);

// Optional outputs of the input projection for a persistent step (B*H <= 64 rows,
// w a multiple of 64): the first adaptive norm's p[row, n] = bf16((1 + scale[row*ldm + n]) x),
// the rows' sums of squares per 64-column tile sumsq[(n/64)*64 + row], and bf16 copies
// cvt_out[c][row][n] = bf16(cvt_in[row*cvt_ld + c*cvt_stride + n]) for c < cvt_chunks.
// p = NULL: none of these.
// First adaptive norm of the persistent step (B*H <= 64 rows): p = bf16((1 + scale) x)
// and the bf16 shift copies (chunk c at cvt_out + c * 64 * w) in 32-column tiles
// [w/32][64 rows][32]; sumsq[(n / 64) * 64 + row] the 64-column tiles' sums of squares.
struct InProjNorm {
  const float* scale; int ldm;
  bf16_t* p;
  float* sumsq;
  const float* cvt_in; int cvt_ld, cvt_stride, cvt_chunks;
  bf16_t* cvt_out;
};

// Input projection in logical slot order: x[e*H+i, n] = W_in[n,:] . X[e, (t+i) mod H, :] + b_in[n],
// with the weights given transposed (w_inT[d, n] = W_in[n, d]); t = NULL: X is a chunk
// already in logical order (row i of env e).  The offset MLP's hidden layer likewise takes
// t = NULL for context age 0.
// The offset conditioning of a few envs in one launch (bf16 models): delta_e as for
// launch_delta_hidden, h1 = bf16(silu(wd1 delta_e + bd1)), d = wd2 h1 + bd2 (wd2 bf16
// [w, w]), cond[e*H + i, n] = bf16(silu(ctau[r, n] + d[n])) with r as for
// launch_cond_expand.  w <= 2048, a multiple of 8; H <= 128.
hipError_t launch_offset_cond(const int64_t* t, const int64_t* t_obs, const int64_t* ages, int B, int H,
                              float delta_bias, const float* wd1, const float* bd1, const bf16_t* wd2,
                              const float* bd2, int w, const float* ctau, int tau_row, bf16_t* cond,
                              hipStream_t s);
// launch_offset_cond (rolling step: ages and tau_row unused) and launch_in_proj (ring
// in slot order from the step counter t, no offset input) in one launch, the input
// projection writing x and the rows' per-64-column sums of squares (sumsq[tile][64])
// only: the first norm's p and shift copies then come from the modulation GEMM
// (GemmArgs nrm_*).  B * H <= 64, w a multiple of 64.
hipError_t launch_offset_cond_in_proj(const int64_t* t, const int64_t* t_obs, int B, int H, float delta_bias,
                                      const float* wd1, const float* bd1, const bf16_t* wd2, const float* bd2, int w,
                                      const float* ctau, bf16_t* cond, const float* X, int D, const float* w_inT,
                                      const float* b_in, float* x, float* sumsq, hipStream_t s);

// dval: NULL, or [B] offsets delta_e concatenated to every slot's input: w_inT then has
// D + 1 rows and row D multiplies delta_e.
hipError_t launch_in_proj(const float* X, const int64_t* t, int B, int H, int D, const float* w_inT,
                          const float* b_in, int w, float* x, const InProjNorm& nrm, const double* dval,
                          hipStream_t s);
// The norm operands of InProjNorm (p, sums of squares, shift copies; nrm.p required)
// for rows x [BH, w] produced by other kernels.  BH <= 64, w a multiple of 64.
hipError_t launch_norm_operands(const float* x, int BH, int w, const InProjNorm& nrm, hipStream_t s);

// Rotary position embedding of the buffer rows' self-attention queries and keys, in place:
// row e*H + i of qkv (row stride ld) holds nq query heads then nkv key heads of hd columns;
// in each, the pair (d, d + hd/2) turns by the angle whose cosine and sine are
// cs[(i * hd/2 + d) * 2 + {0, 1}] (slot i's table row).
template <typename T>
hipError_t launch_rope(T* qkv, int ld, int BH, int H, int nq, int nkv, int hd, const float* cs, hipStream_t s);

// dval[e] = p_e / H + delta_bias (float64) with p_e = ages[e], or *t - t_obs[e], or 0 (no step counter).
hipError_t launch_offset_value(const int64_t* t, const int64_t* t_obs, const int64_t* ages, int B, int H,
                               float delta_bias, double* dval, hipStream_t s);
// Inputs of the DynamicVLA-style offset form, row = e*H + i in logical order, emb the
// flow-time sinusoid (launch_time_embedding's, evaluated in float64):
//   mode 0, the action-time MLP: z[row] = [x[row] ; emb(tau) ; dval[e] ; 0 ...] up to ldz,
//           tau = (i + 1) / H, or (tau_row + 1) / tau_den for every slot when tau_row >= 0;
//   mode 1, the offset adapter:  z[row] = [x[row] ; emb(dval[e])] (columns >= 2w zero).
template <typename T>
hipError_t launch_offset_rows(int mode, const float* x, const double* dval, int B, int H, int w, int tau_row,
                              int tau_den, T* z, int ldz, hipStream_t s);

// Analytic velocity fields (logical order): OT v = (x - a*)/tau, LINEAR v = lambda x, with
// tau = tau_i = (i+1)/H of the ring (rotated by t), or tau_all for every slot of a chunk
// (t = NULL: X in logical order).
// With state (relative actions, [B, D] with mask [D] of 0/1), the OT field's absolute target
// a* is aimed at as a* - mask * state.
hipError_t launch_analytic_velocity(int kind, const float* X, const int64_t* t, int B, int H, int D,
                                    const float* param, float tau_all, const float* state, const float* mask,
                                    float* v, hipStream_t s);

// Relative actions: X[e, (t+i) mod H, :] += (1 - tau_i) mask * (s_prev[e] - state[e]) unless
// has_prev[e] is 0 (the env's first step), then s_prev[e] = state[e], has_prev[e] = 1.
hipError_t launch_relative_shift(float* X, const int64_t* t, int B, int H, int D, const float* mask,
                                 const float* state, float* s_prev, int* has_prev, hipStream_t s);

// Euler step of a full-horizon chunk: X[e, i, :] -= dt * v[e*H + i, :].
hipError_t launch_euler_chunk(float* X, const float* v, int B, int H, int D, float dt, hipStream_t s);

// Euler update of every slot, release of logical slot 0 into action[e,:] (plus mask * state[e]
// when state is given: relative dimensions released in absolute coordinates), Philox
// noise for action index r = t + H into the released physical slot, t += 1.  One block per
// env; ticket is a device word that is zero between launches (the last block re-arms it).
hipError_t launch_euler_release(float* X, const float* v, int64_t* t, int B, int H, int D,
                                uint64_t seed, float* action, unsigned* ticket, const float* state,
                                const float* mask, const int* err, int* host_flag, hipStream_t s);

// Zero n 32-bit words on stream s with a kernel.
hipError_t launch_zero_u32(unsigned* p, long long n, hipStream_t s);

// Fill X[e, r mod H, :] with the Philox noise of action r, for r = 0..H-1.
hipError_t launch_ring_init(float* X, int B, int H, int D, uint64_t seed, hipStream_t s);

// Sinusoidal flow-time embedding of tau_i = (i+1)/H: emb[i, j] = sin(1000 tau w_j),
// emb[i, w/2 + j] = cos(1000 tau w_j), w_j = 10000^(-j/(w/2)); evaluated in float64.
template <typename T>
hipError_t launch_time_embedding(int H, int w, T* emb, hipStream_t s);

template <typename T>
hipError_t launch_convert(const float* src, T* dst, long long n, hipStream_t s);

// Context publication: for i < n: slot[env[i]] = new_slot[i]; t_obs[env[i]] = tobs[i].
struct PublishBatch {
  int n;
  int env[32];
  int new_slot[32];
  long long tobs[32];
};
hipError_t launch_publish(const PublishBatch& pb, int* slot, int64_t* t_obs, hipStream_t s);

// NaN/Inf scan used by the debug mode: flag[0] |= any non-finite value.
hipError_t launch_check_finite(const float* p, long long n, int* flag, hipStream_t s);
template <typename T>
hipError_t launch_check_finite_t(const T* p, long long n, int* flag, hipStream_t s);

}  // namespace ravel
