// Phase list of the persistent few-row step (internal to the library).
#pragma once

#include "kernels.h"

namespace ravel {

enum PhaseType : int { PH_GEMM = 2, PH_ATTN = 3, PH_ROPE = 4 };

// GEMM activation operand
enum PAMode : int {
  PA_BF16 = 0,  // A[m][k] in bf16
  // adaptive RMSNorm applied on load: h[m][k] = r[m] * p[m][k] + shift[m][k] (shift optional), with
  // p = bf16((1 + scale) * x) written by whoever produced the residual x, and
  // r[m] = 1 / sqrt(mean_k x[m][k]^2 + eps) from the per-64-column row sums of squares of x
  PA_NORM = 1,
  // the FOP cross-attention output of one head, computed by the item itself from
  // the adapter queries A = qa (bf16): the item's K range is exactly one head
  // (hd = 256, kw = 1), the head's keys and values are rows [x_nf][x_ld] of
  // xk / xv (x_nf <= 16) at column (head / x_group) * 256, scores scaled by x_scale
  PA_XATTN = 2,
};
enum PEMode : int { PE_BF16 = 0, PE_F32 = 1, PE_GEGLU = 2, PE_RESID = 3 };
// scale of the next norm, applied to a new residual x to form p: per (row, column)
// modulation rows, or one vector over columns
enum NSMode : int { NS_ROW = 0, NS_COL = 1 };

// Grid barrier: kBarrierGroups group counters (one 256-byte line each), a top
// counter, a generation word and an exit counter; 64 * (3 + groups) words.
constexpr int kBarrierGroups = 32;
constexpr int kBarrierWords = 64 * (3 + kBarrierGroups);
// polls (each a device-coherent load) before a barrier gives up and flags an
// error: seconds, far above any phase of a step
constexpr int kBarrierSpinLimit = 1 << 22;
// split-K ranges per output tile (a GEMM item covers 256 * kw of K, kw in {1, 2};
// kw = 2 only for plain bf16 activations)
constexpr int kMaxKSplit = 8;
// key splits of one attention (env, head)
constexpr int kMaxAttnSplit = 32;
// keys of one attention split: 32 KB of keys and values (a split's share is
// fetched into registers, 128 bytes per thread, while the block waits at the
// barrier that opens the phase)
__host__ __device__ constexpr int attn_keys_per_split_max(int hd) { return (8192 / hd) < 256 ? (8192 / hd) : 256; }

// Activations produced inside the launch are written once per launch (each phase
// has its own output buffers) and every 128-byte line of them by exactly one block,
// so the phases after it read them with plain loads, shared through each XCD's L2;
// a_coh = 1 keeps device-coherent loads for an operand whose lines are shared by
// several writers (attention outputs of heads narrower than 64 dims).
struct PGemm {
  int a_mode, e_mode;  // PAMode, PEMode
  int kw, ksplit;      // K per item = 256 * kw; items = tiles(N, 64) * ksplit
  int M, N, K;
  const bf16_t* A; int lda;            // PA_BF16: A; PA_NORM: p
  int a_t32;                           // PA_BF16: A stored in 32-column tiles [K/32][64 rows][32]
  int a_coh;                           // 1: device-coherent loads of A
  const bf16_t* shift; int ld_shift;   // PA_NORM: bf16 shift rows or NULL
  int sh_t32;                          // PA_NORM: shift in 32-column tiles [K/32][64 rows][32]
  // PA_NORM: row sums of squares of x per 64-column tile, entry (t, row) at
  // sumsq_in[(t * 64 + row) * sq_in_ld]
  const float* sumsq_in; int sq_in_ld; float eps;
  const bf16_t* W; int ldw;            // weights [N][ldw]
  const float* bias;                   // PE_F32 (or NULL)
  bf16_t* out_t; int ldo;              // PE_BF16 / PE_GEGLU
  int out_t32;                         // PE_GEGLU: output in 32-column tiles [N/64][64 rows][32]
  float* out_f; int ldof;              // PE_F32 output, or the new residual x (PE_RESID)
  const float* x_in;                   // PE_RESID: the residual x before the update (stride ldof)
  const float* gate; int ldg;          // PE_RESID: gate rows, or NULL and then
  const float* gate_scalar;            // tanh(*gate_scalar)
  int ns_mode; const float* ns; int ldns;  // PE_RESID: scale of the next norm
  bf16_t* p_out; int ldp;              // PE_RESID: p of the next norm
  int p_t32;                           // PE_RESID: p in 32-column tiles [N/32][64 rows][32]
  // PE_RESID: row sums of squares of the new x, entry (tile, row) at
  // sumsq_out[(tile * 64 + row) * sq_out_ld] (32: one 128-byte line per entry)
  float* sumsq_out; int sq_out_ld;
  float* partial; unsigned* counters;  // split-K partial tiles, per-tile tickets
  // 1: the ksplit blocks of a tile meet and each finishes a slice of its rows
  // (needs one item per block); 0: the last block to arrive finishes the tile
  int coop;
  const bf16_t* xk; const bf16_t* xv;  // PA_XATTN: FOP keys and values of the adapter
  int x_ld, x_nf, x_group;
  float x_scale;
  // whole-K items (wk = column blocks of 16 per item, 1 or 2; 0: K ranges of 256 * kw
  // with split tiles): item t covers columns [16 wk t, 16 wk (t + 1)) over the whole K,
  // wave w its K quarter [w K/4, (w + 1) K/4) (K/4 a multiple of 32, at most 256); the
  // quarters are added through LDS, so no tile is split across blocks.  PA_NORM
  // operands with p and shift in 32-column tiles (plain loads), PE_BF16 / PE_GEGLU
  // (wk = 2: a 16-column gate block and its up block) / PE_F32 epilogues.
  int wk;
};

// Rotary positions (the rows' queries and keys written by the phase before): item =
// one row e*H + i of qkv (row stride ld), whose nh = nq + nkv heads of hd columns
// each turn their pairs (d, d + hd/2) by the angle with cosine cs[(i * hd/2 + d) * 2]
// and sine cs[(i * hd/2 + d) * 2 + 1], written to the same place of out (a buffer of
// the same layout); hd % 8 == 0.
struct PRope {
  const bf16_t* qkv; bf16_t* out; int ld;
  int coh;  // 1: device-coherent loads of qkv (written by whole-K items in 16-column pieces)
  int H, nh, hd;
  const float* cs;
};

// Side work of a phase, run by its blocks that have no item of their own: items
// item0 .. item0 + nitems - 1 of a modulation GEMM out = A W^T + bias over the whole
// K (32 output columns per item, M <= 64 rows, A row-major bf16), fp32 out rows, and
// for the columns of up to two shift ranges [shift_col[s], shift_col[s] + shift_w)
// also bf16 copies in 32-column tiles [shift_w/32][64 rows][32] at shift_out[s].
struct PSide {
  const bf16_t* A; int lda;
  const bf16_t* W; int ldw;
  const float* bias;
  float* out; int ldo;
  bf16_t* shift_out[2]; int shift_col[2]; int shift_w;
  int M, N, K;
  int item0, nitems;
};

struct alignas(16) Phase {
  int type, items, pad0, pad1;
  union {
    PGemm g;
    AttnArgs at;
    PRope r;
  };
  PSide side;
};

// env_slot: [nenv] active context slot per env (read once per launch).
// times: optional [nphase + 1] wall-clock stamps taken by block 0 at the start,
// after each phase's barrier, and at its end (NULL: none).
// counters: the ncounters split counters (one per kCounterStride words) that the
// phases' tiles and heads use, each once per launch; zero at the launch, and zeroed
// again by the last block to leave it.
hipError_t launch_persistent(const Phase* phases, int nphase, const int* env_slot, int nenv, int mt, int hd, int blocks,
                             unsigned* bar, int* err, unsigned long long* times, unsigned* counters, int ncounters,
                             hipStream_t s);
// Blocks of the persistent kernel (row tiles mt, head dimension hd) that can be
// co-resident (0 on error).
int persistent_max_blocks(int mt, int hd);

}  // namespace ravel
