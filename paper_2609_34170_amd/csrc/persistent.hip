// Persistent few-row step: the transformer layers of a batch whose B*H rows fit
// one 64-row MFMA tile (B*H <= 64, e.g. one env with 50 slots) run inside ONE
// kernel (one block per CU, all co-resident) that walks a host-built list of
// phases separated by hierarchical grid barriers.
//
// At these sizes every phase is a chain of memory round trips rather than a
// bandwidth problem, so the kernel is laid out to keep that chain short:
//  * the descriptor of phase p + 2 and the weight fragments of this block's
//    first item of phase p + 1 are fetched while the block waits at barrier
//    p + 1 (weights and descriptors never change during a launch);
//  * every load of an item is issued before the first of them is used (no
//    loops whose trip counts hide loads behind one another);
//  * one thread per block performs the device-scope acquire after a barrier
//    or a split ticket, and every wave drains its stores before arriving.
//
// Phases (the input projection, launched before, writes the first norm's
// operands):
//  * GEMM: an item is a 64-column tile times a K range of 256 * kw; the four
//    waves take K quarters and are reduced through LDS; the activation operand
//    is bf16, or normalised on load as h = r * p + shift with r = 1/rms(x)
//    from the row sums; split-K ranges are added in fixed order by the last
//    block to arrive at the tile's ticket, whose epilogue writes bf16 / fp32
//    outputs, gelu(gate) * up, or a gated residual update of x that also
//    writes the next norm's p and the new row sums of squares; a K of at most
//    1024 that the output tiles would split across blocks is instead covered
//    whole by items of 16 (GeGLU: 2 x 16) columns, which need no meet;
//  * ATTN: an item is one (env, head, key split): its keys and values are
//    staged in LDS in one batch, the four waves take 16 queries each, and the
//    splits are merged by the last item of the (env, head) to arrive.
// Values handed to another block are written with device-coherent stores and
// read with device-coherent (sc1) buffer loads, which bypass the CU's L1 and are
// served by the L2, coherent across the XCDs on this part: measured with a
// stale-read probe (one block rewrites a buffer before each barrier, every block
// counts stale values after it, with the L1 pre-filled by plain reads) -- zero
// stale values out of 10^9 -- so no cache-invalidating acquire is needed after a
// barrier or ticket (an agent-scope acquire invalidates the L2 and costs ~2 us
// per phase).  Data written before the launch (weights, modulation, context) is
// read with plain loads.  Producers drain their stores before arriving at a
// barrier or ticket.  Spins are bounded: a barrier that does not complete sets
// the error flag and every wave exits.
#include "kernels.h"
#include "persistent.h"

namespace ravel {
namespace {

template <int HD>
struct AttnCfg {
  static constexpr int KPS = attn_keys_per_split_max(HD);  // keys staged per split
  static constexpr int KLD = HD + 8;                       // K row stride in LDS
  static constexpr int VLD = KPS + 8;                      // V^T row stride in LDS
  static constexpr int ELEMS = KPS * KLD + HD * VLD;
};
constexpr int cmax(int a, int b) { return a > b ? a : b; }
constexpr int kAttnElems =
    cmax(cmax(AttnCfg<32>::ELEMS, AttnCfg<64>::ELEMS), cmax(AttnCfg<128>::ELEMS, AttnCfg<256>::ELEMS));

struct PSmem {
  union {
    float red[4][16][64][4];  // GEMM: per-wave partial tiles
    bf16_t at[kAttnElems];    // attention: K rows, then V^T
    struct {
      float ml[kMaxAttnSplit][64][2];  // attention merge: (max, sum) per split and query
      float wgt[kMaxAttnSplit][64];    // merge weights
    } mg;
    // whole-K GEMM: the norm's shift fragments, staged by direct-to-LDS loads, wave w's
    // fragment (i, f) at shs[w][i * 8 + f] in lane order
    u32x4_t shs[4][32][64];
  };
  float rscale[64];
  float rowsq[64][17];
  bf16_t xvt[256 * 20];  // PA_XATTN: the head's FOP values transposed, [dim][key], row stride kXLD
  int flag;
};
constexpr int kXLD = 20;

RAVEL_DEV int uni(int x) { return __builtin_amdgcn_readfirstlane(x); }

// Loads go through buffer resources on wave-uniform bases with per-lane byte
// offsets.  A lane with nothing to load passes an offset past the resource's
// range and reads zeros: no branch around the load, so a batch of predicated
// loads stays in flight together (a load under a branch that also writes its
// register on the other path makes the compiler wait for it at once).
// PLAIN: data written before the launch.  COH: data written during the launch,
// device-coherent (sc1: bypasses the CU's L1, served by the coherent L2).
typedef __amdgpu_buffer_rsrc_t rsrc_t;
constexpr int PLAIN = 0, COH = 16;
constexpr unsigned kOutOfRange = 0x80000000u;
RAVEL_DEV rsrc_t rsrc(const void* base) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, 0x7fffffff, 0x00020000);
}
RAVEL_DEV int boff(bool ok, size_t byte_off) { return (int)(ok ? (unsigned)byte_off : kOutOfRange); }
template <int AUX>
RAVEL_DEV u32x4_t ld16(rsrc_t r, int off) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, AUX);
}
template <int AUX>
RAVEL_DEV f32x4_t ld_f4(rsrc_t r, int off) {
  const u32x4_t v = ld16<AUX>(r, off);
  return *reinterpret_cast<const f32x4_t*>(&v);
}
template <int AUX>
RAVEL_DEV bf16x8_t ld_b8(rsrc_t r, int off) {
  const u32x4_t v = ld16<AUX>(r, off);
  return *reinterpret_cast<const bf16x8_t*>(&v);
}
template <int AUX>
RAVEL_DEV float ld_f1(rsrc_t r, int off) {
  return __uint_as_float(__builtin_amdgcn_raw_buffer_load_b32(r, off, 0, AUX));
}
template <int AUX>
RAVEL_DEV float2 ld_f2(rsrc_t r, int off) {
  const auto v = __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, AUX);
  return float2{__uint_as_float(v[0]), __uint_as_float(v[1])};
}
// device-coherent stores (sc1 buffer stores: what a relaxed agent-scope atomic
// store lowers to, but widened to 16 bytes and issued as global accesses)
RAVEL_DEV void st_f4(rsrc_t r, size_t byte_off, f32x4_t v) {
  __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4_t, v), r, (int)byte_off, 0, COH);
}
RAVEL_DEV void st_f1(rsrc_t r, size_t byte_off, float v) {
  __builtin_amdgcn_raw_buffer_store_b32(__float_as_uint(v), r, (int)byte_off, 0, COH);
}
RAVEL_DEV void st_bf16x4(rsrc_t r, size_t byte_off, float v0, float v1, float v2, float v3) {
  const u32x2_t w = {pack_bf16x2(v0, v1), pack_bf16x2(v2, v3)};
  __builtin_amdgcn_raw_buffer_store_b64(w, r, (int)byte_off, 0, COH);
}
// four fp16 values (round to nearest even), and their load back to fp32
typedef __attribute__((__vector_size__(4 * sizeof(_Float16)))) _Float16 f16x4_t;
RAVEL_DEV void st_f16x4(rsrc_t r, size_t byte_off, f32x4_t v) {
  const f16x4_t h = __builtin_convertvector(v, f16x4_t);
  __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(u32x2_t, h), r, (int)byte_off, 0, COH);
}
template <int AUX>
RAVEL_DEV f32x4_t ld_f16x4(rsrc_t r, int off) {
  const u32x2_t v = __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, AUX);
  return __builtin_convertvector(__builtin_bit_cast(f16x4_t, v), f32x4_t);
}

// threadIdx.x behind an empty asm: index arithmetic derived from it stays inside
// the work item that needs it instead of being hoisted out of the phase loop,
// where the invariants of every item kind would stay live for the whole kernel
RAVEL_DEV int local_tid() {
  int t = threadIdx.x;
  asm volatile("" : "+v"(t));
  return t;
}

// A copy of a descriptor held in LDS, with every word made wave-uniform.
template <class T>
RAVEL_DEV T make_uniform(const T& s) {
  static_assert(sizeof(T) % 4 == 0, "descriptor size");
  T d;
  const int* si = reinterpret_cast<const int*>(&s);
  int* di = reinterpret_cast<int*>(&d);
#pragma unroll
  for (int i = 0; i < (int)(sizeof(T) / 4); ++i) di[i] = __builtin_amdgcn_readfirstlane(si[i]);
  return d;
}


// Split tiles and split heads count their arrivals in counters of their own: every
// phase has a range of counters used once per launch (zeroed by the last block to
// leave the launch), so no block waits to re-arm one.
//
// Ticket of a split tile / split attention head: every wave drains its stores,
// thread 0 takes the ticket.
RAVEL_DEV bool last_arrival(unsigned* counter, unsigned arrivals, int* s_flag) {
  wait_memory();
  __syncthreads();
  if (threadIdx.x == 0) {
    const unsigned prev = __hip_atomic_fetch_add(gptr(counter), 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    *s_flag = prev == arrivals - 1;
  }
  __syncthreads();
  return *s_flag != 0;
}

// Meeting point of the blocks of one split tile / split head (each holds one
// item of the phase, so all of them are running): every wave drains its stores,
// thread 0 arrives and polls until all have arrived (bounded; on timeout the
// error flag is set and false returned).
RAVEL_DEV bool group_meet(unsigned* counter, unsigned arrivals, int* err, int* s_flag) {
  wait_memory();
  __syncthreads();
  if (threadIdx.x == 0) {
    int ok = 1;
    __hip_atomic_fetch_add(gptr(counter), 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    int spins = 0;
    while (__hip_atomic_load(gptr(counter), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < arrivals) {
      __builtin_amdgcn_s_sleep(1);
      if (++spins > kBarrierSpinLimit) {
        __hip_atomic_fetch_or(gptr(err), 2, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        ok = 0;
        break;
      }
      // another block gave up: leave instead of waiting out the limit
      if ((spins & 255) == 0 && __hip_atomic_load(gptr(err), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) {
        ok = 0;
        break;
      }
    }
    *s_flag = ok;
  }
  __syncthreads();
  return *s_flag != 0;
}

// Hierarchical grid barrier, split in two so that loads can be issued between
// arrival and wait.  Group g's counter sits on its own 256-byte line; the last
// arrival of a group bumps the top counter and the last top arrival publishes
// the generation word every block polls (polling the top counter itself instead
// is slower: the polls delay the group arrivals on that line).
RAVEL_DEV void barrier_arrive(unsigned* bar, unsigned gen) {
  const int G = kBarrierGroups;
  const int g = blockIdx.x % G;
  const unsigned per = (gridDim.x - g + G - 1) / G;
  const unsigned prev = __hip_atomic_fetch_add(gptr(bar + 64 * (1 + g)), 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  if (prev == gen * per - 1) {
    const unsigned t = __hip_atomic_fetch_add(gptr(bar + 64 * (1 + G)), 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (t == gen * (unsigned)G - 1) __hip_atomic_store(gptr(bar), gen, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

RAVEL_DEV int barrier_wait(unsigned* bar, unsigned gen, int* err) {
  int spins = 0;
  while (__hip_atomic_load(gptr(bar), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) < gen) {
    __builtin_amdgcn_s_sleep(1);
    if (++spins > kBarrierSpinLimit) {
      __hip_atomic_fetch_or(gptr(err), 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      return 0;
    }
    // another block gave up (a barrier or a split meeting timed out): leave now
    if ((spins & 255) == 0 && __hip_atomic_load(gptr(err), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) return 0;
  }
  return 1;
}

// ---------------------------------------------------------------------------
// GEMM
// ---------------------------------------------------------------------------
// Weight fragments of an item: wave w holds rows n0 + 16c + (lane & 15) and the
// K range kb + 32f + 8(lane >> 4) .. +7 for its quarter of the item's K range.
template <int KW>
RAVEL_DEV void load_w(const PGemm& g, int item, u32x4_t (&wf)[16]) {
  const int tid = local_tid();
  const int lane = tid & 63, wave = tid >> 6, l16 = lane & 15, grp = lane >> 4;
  const int tiles = (g.N + 63) >> 6, tile = item % tiles, z = item / tiles;
  const int n0 = tile * 64, kb = z * 256 * KW + wave * 64 * KW;
  const rsrc_t rw = rsrc(g.W);
#pragma unroll
  for (int f = 0; f < 4; ++f) {
    const int k = kb + f * 32 + grp * 8;
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int n = n0 + c * 16 + l16;
      wf[c * 4 + f] = ld16<PLAIN>(rw, boff(f < 2 * KW && n < g.N && k < g.K, ((size_t)n * g.ldw + k) * 2));
    }
  }
}

// PA_XATTN weight fragments: the same rows, with the K slots of lane group grp
// holding dims 32f + 4grp .. +3 and 32f + 16 + 4grp .. +3 of the wave's quarter --
// the order in which the item's attention output leaves its MFMAs.
RAVEL_DEV void load_w_xattn(const PGemm& g, int item, u32x4_t (&wf)[16]) {
  const int tid = local_tid();
  const int lane = tid & 63, wave = tid >> 6, l16 = lane & 15, grp = lane >> 4;
  const int tiles = (g.N + 63) >> 6, tile = item % tiles, z = item / tiles;
  const int n0 = tile * 64, kb = z * 256 + wave * 64;
  const rsrc_t rw = rsrc(g.W);
#pragma unroll
  for (int f = 0; f < 4; ++f) {
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int n = n0 + c * 16 + l16;
      const bool ok = f < 2 && n < g.N;
      const int k = kb + f * 32 + grp * 4;
      const auto lo = __builtin_amdgcn_raw_buffer_load_b64(rw, boff(ok && k < g.K, ((size_t)n * g.ldw + k) * 2), 0, PLAIN);
      const auto hi =
          __builtin_amdgcn_raw_buffer_load_b64(rw, boff(ok && k + 16 < g.K, ((size_t)n * g.ldw + k + 16) * 2), 0, PLAIN);
      wf[c * 4 + f] = u32x4_t{lo[0], lo[1], hi[0], hi[1]};
    }
  }
}

// Whole-K item fragments: wave w holds rows n0 + 16c + (lane & 15), c < wk, and the
// K range w K/4 + 32f + 8(lane >> 4) .. +7, f < K/128 (fragment c * 8 + f).
RAVEL_DEV void load_w_wk(const PGemm& g, int item, u32x4_t (&wf)[16]) {
  const int tid = local_tid();
  const int lane = tid & 63, wave = tid >> 6, l16 = lane & 15, grp = lane >> 4;
  const int n0 = item * 16 * g.wk, kq = g.K >> 2, kb = wave * kq;
  const rsrc_t rw = rsrc(g.W);
#pragma unroll
  for (int c = 0; c < 2; ++c)
#pragma unroll
    for (int f = 0; f < 8; ++f) {
      const int n = n0 + c * 16 + l16, k = kb + f * 32 + grp * 8;
      wf[c * 8 + f] = ld16<PLAIN>(rw, boff(c < g.wk && f * 32 < kq && n < g.N, ((size_t)n * g.ldw + k) * 2));
    }
}

RAVEL_DEV void load_weights(const PGemm& g, int item, u32x4_t (&wf)[16]) {
  if (g.wk)
    load_w_wk(g, item, wf);
  else if (g.a_mode == PA_XATTN)
    load_w_xattn(g, item, wf);
  else if (g.kw == 2)
    load_w<2>(g, item, wf);
  else
    load_w<1>(g, item, wf);
}

// Rows of a cooperative split-K tile that block z finishes: [z * rp, (z + 1) * rp)
// with rp even, so that two rows sharing a 128-byte line of a 32-column-tile
// output go to one block.
RAVEL_DEV int coop_rows(const PGemm& g) {
  const int rp = (g.M + g.ksplit - 1) / g.ksplit;
  return (rp + 1) & ~1;
}
// Byte offset of A[m][k] (bf16): row-major with stride lda, or 32-column tiles.
RAVEL_DEV size_t a_off(const PGemm& g, int m, int k) {
  return g.a_t32 ? ((size_t)(k >> 5) * 2048 + (size_t)m * 32 + (k & 31)) * 2 : ((size_t)m * g.lda + k) * 2;
}
// Byte offset of element (m, k) of a bf16 matrix in 32-column tiles [K/32][64 rows][32].
RAVEL_DEV size_t t32_off(int m, int k) { return ((size_t)(k >> 5) * 2048 + (size_t)m * 32 + (k & 31)) * 2; }
// Byte offset of shift[m][k] (bf16): row-major with stride ld_shift, or 32-column tiles.
RAVEL_DEV size_t sh_off(const PGemm& g, int m, int k) {
  return g.sh_t32 ? ((size_t)(k >> 5) * 2048 + (size_t)m * 32 + (k & 31)) * 2 : ((size_t)m * g.ld_shift + k) * 2;
}
// Byte offset of p_out[m][n] (bf16) of a residual update.
RAVEL_DEV size_t p_off(const PGemm& g, int m, int n) {
  return g.p_t32 ? ((size_t)(n >> 5) * 2048 + (size_t)m * 32 + (n & 31)) * 2 : ((size_t)m * g.ldp + n) * 2;
}
// Activation fragments af[i][f] of a split item (rows i*16 + (lane & 15), K range
// kb + 32f + 8(lane >> 4) .. +7), with cache policy AUX.
template <int AUX, int MT, int NF>
RAVEL_DEV void load_a_frags(const PGemm& g, rsrc_t rA, int kb, bf16x8_t (&af)[MT][NF]) {
  const int lane = local_tid() & 63, l16 = lane & 15, grp = lane >> 4;
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int f = 0; f < NF; ++f) {
      const int m = i * 16 + l16, k = kb + f * 32 + grp * 8;
      af[i][f] = ld_b8<AUX>(rA, boff(m < g.M && k < g.K, a_off(g, m, k)));
    }
}
// Byte offset of output column c (of N / 2) of row m of a gated-GeLU phase.
RAVEL_DEV size_t geglu_off(const PGemm& g, int m, int c) {
  return g.out_t32 ? ((size_t)(c >> 5) * 2048 + (size_t)m * 32 + (c & 31)) * 2 : ((size_t)m * g.ldo + c) * 2;
}

// Epilogue operands of one slot of a cooperative split-K tile: residual x,
// gate, next norm scale, bias (loaded at the start of the item, long before the
// split meets).
struct CoopOps {
  f32x4_t ex, eg, es, eb;
};
template <int MT>
RAVEL_DEV CoopOps coop_operands(const PGemm& g, int tile, int z, int s0, bool use);
template <int MT>
RAVEL_DEV void coop_epilogue(const PGemm& g, int tile, int z, int tiles, PSmem& sm, const CoopOps& first);

// PA_XATTN: the item's activation operand is head z's cross-attention output
// o = softmax(q k^T * scale) v over the FOP tokens, computed here from the query
// fragments af (this wave's 64 dims of the head, rows i*16 + l16).  Each wave
// forms its partial scores S^T = K Q^T over its dims; the four partials are added
// through LDS in wave order; each lane then holds rows l16 and keys 4grp .. +3, the
// row softmax is reduced over the four lane groups, and P^T (bf16) feeds
// O^T = V^T P^T (16x16x16 MFMAs, V^T staged transposed in LDS) for the wave's
// four 16-dim tiles.  The normalised outputs become the GEMM's B fragments in
// the K-slot order of load_w_xattn.  Templated on the KW = 1 fragment shape.
template <int MT>
RAVEL_DEV void xattn_operands(const PGemm& g, const bf16x8_t (&xkf)[2], const u32x4_t (&xvc)[2],
                              bf16x8_t (&af)[MT][2], PSmem& sm) {
  typedef __attribute__((ext_vector_type(4))) short s16x4_t;
  const int tid = local_tid(), lane = tid & 63, wave = tid >> 6;
  const int l16 = lane & 15, grp = lane >> 4;
  f32x4_t sp[MT];
#pragma unroll
  for (int i = 0; i < MT; ++i) {
    sp[i] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int f = 0; f < 2; ++f) sp[i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(xkf[f], af[i][f], sp[i], 0, 0, 0);
  }
  __syncthreads();  // LDS may still be read by this block's previous item
#pragma unroll
  for (int i = 0; i < MT; ++i) *(f32x4_t*)&sm.red[wave][i][lane][0] = sp[i];
#pragma unroll
  for (int r = 0; r < 2; ++r) {
    const int c = tid + r * 256, key = c >> 5, d0 = (c & 31) * 8;
    const bf16_t* h = reinterpret_cast<const bf16_t*>(&xvc[r]);
#pragma unroll
    for (int j = 0; j < 8; ++j) sm.xvt[(d0 + j) * kXLD + key] = h[j];
  }
  __syncthreads();
  const float sl2 = g.x_scale * 1.4426950408889634f;
  s16x4_t pb[MT];
  float inv[MT];
#pragma unroll
  for (int i = 0; i < MT; ++i) {
    f32x4_t s = *(const f32x4_t*)&sm.red[0][i][lane][0];
#pragma unroll
    for (int w = 1; w < 4; ++w) {
      const f32x4_t t = *(const f32x4_t*)&sm.red[w][i][lane][0];
      s[0] += t[0];
      s[1] += t[1];
      s[2] += t[2];
      s[3] += t[3];
    }
    float x[4], mx = -INFINITY;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      x[r] = grp * 4 + r < g.x_nf ? s[r] * sl2 : -INFINITY;
      mx = fmaxf(mx, x[r]);
    }
    mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
    float p[4], l = 0.f;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      p[r] = __builtin_amdgcn_exp2f(x[r] - mx);
      l += p[r];
    }
    l += __shfl_xor(l, 16, 64);
    l += __shfl_xor(l, 32, 64);
    inv[i] = 1.f / l;
    const u32x2_t pw = {pack_bf16x2(p[0], p[1]), pack_bf16x2(p[2], p[3])};
    pb[i] = __builtin_bit_cast(s16x4_t, pw);
  }
#pragma unroll
  for (int f = 0; f < 2; ++f) {
    f32x4_t ot[2][MT];
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int d = wave * 64 + (2 * f + h) * 16 + l16;
      const s16x4_t vf = __builtin_bit_cast(s16x4_t, *(const u32x2_t*)&sm.xvt[d * kXLD + grp * 4]);
#pragma unroll
      for (int i = 0; i < MT; ++i)
        ot[h][i] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(vf, pb[i], f32x4_t{0.f, 0.f, 0.f, 0.f}, 0, 0, 0);
    }
#pragma unroll
    for (int i = 0; i < MT; ++i) {
      const float r = inv[i];
      const u32x4_t w = {pack_bf16x2(ot[0][i][0] * r, ot[0][i][1] * r), pack_bf16x2(ot[0][i][2] * r, ot[0][i][3] * r),
                         pack_bf16x2(ot[1][i][0] * r, ot[1][i][1] * r), pack_bf16x2(ot[1][i][2] * r, ot[1][i][3] * r)};
      af[i][f] = __builtin_bit_cast(bf16x8_t, w);
    }
  }
}

template <int MT, int KW, class AfterLoads>
RAVEL_DEV void gemm_item(const PGemm& g, int item, const u32x4_t (&w16)[16], int* err, PSmem& sm,
                         AfterLoads&& after_loads) {
  bf16x8_t wf[4][4];
#pragma unroll
  for (int c = 0; c < 4; ++c)
#pragma unroll
    for (int f = 0; f < 4; ++f) wf[c][f] = __builtin_bit_cast(bf16x8_t, w16[c * 4 + f]);
  constexpr int NF = 2 * KW;
  const int tid = local_tid(), lane = tid & 63, wave = tid >> 6;
  const int l16 = lane & 15, grp = lane >> 4;
  const int tiles = (g.N + 63) >> 6, tile = item % tiles, z = item / tiles;
  const int n0 = tile * 64;
  const int kb = z * 256 * KW + wave * 64 * KW;
  const bool norm = g.a_mode == PA_NORM;
  const bool has_shift = norm && g.shift != nullptr;

  // one batch of loads: the norm's shift rows (written before the launch: plain
  // loads) first, then the activations and the row sums of squares written by the
  // previous phase (coherent loads)
  const rsrc_t rA = rsrc(g.A), rS = rsrc(g.shift);
  bf16x8_t af[MT][NF], sh[MT][NF];
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int f = 0; f < NF; ++f) {
      const int m = i * 16 + l16, k = kb + f * 32 + grp * 8;
      sh[i][f] = ld_b8<PLAIN>(rS, boff(has_shift && m < g.M && k < g.K, sh_off(g, m, k)));
    }
  // (the cache policy is part of the instruction: one batch per policy, chosen by a
  // wave-uniform branch, rather than both loads and a select)
  if (g.a_coh)
    load_a_frags<COH, MT, NF>(g, rA, kb, af);
  else
    load_a_frags<PLAIN, MT, NF>(g, rA, kb, af);
  // PA_XATTN: the head's keys (this wave's 64 dims; lane: key l16) and its values
  // (16-byte chunks c = tid, tid + 256: key c / 32, dims (c % 32) * 8), plain loads
  const bool xattn = g.a_mode == PA_XATTN;
  const int xoff = xattn ? (z / g.x_group) * 256 : 0;
  bf16x8_t xkf[2];
  u32x4_t xvc[2];
  if (xattn) {
    const rsrc_t rK = rsrc(g.xk), rV = rsrc(g.xv);
#pragma unroll
    for (int f = 0; f < 2; ++f)
      xkf[f] = ld_b8<PLAIN>(rK, boff(l16 < g.x_nf, ((size_t)l16 * g.x_ld + xoff + wave * 64 + f * 32 + grp * 8) * 2));
#pragma unroll
    for (int r = 0; r < 2; ++r) {
      const int c = tid + r * 256, key = c >> 5;
      xvc[r] = ld16<PLAIN>(rV, boff(key < g.x_nf, ((size_t)key * g.x_ld + xoff + (c & 31) * 8) * 2));
    }
  }
  float sq[16];
  const int row = tid & 63, part = tid >> 6, nt = g.K >> 6;
  if (norm) {
    const rsrc_t rQ = rsrc(g.sumsq_in);
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      const int t = part + 4 * j;
      sq[j] = ld_f1<PLAIN>(rQ, boff(t < nt && row < g.M, (size_t)(t * 64 + row) * g.sq_in_ld * 4));
    }
  }
  // a cooperative split tile's epilogue operands of this block's first slots
  const CoopOps ops = coop_operands<MT>(g, tile, z, 0, g.ksplit > 1 && g.coop);
  after_loads();
  if constexpr (KW == 1) {
    if (xattn) xattn_operands<MT>(g, xkf, xvc, af, sm);
  }

  // The norm's operand is h = r p + shift (r = 1 / rms(x) per row), so
  // W h = r (W p + W shift / r): the shift product runs while p is in flight,
  // and no bf16 h is formed.  Lane (l16, grp) of fragment (c, i) holds row
  // i*16 + l16, columns n0 + 16c + 4grp .. +3.
  f32x4_t acc[4][MT];
#pragma unroll
  for (int c = 0; c < 4; ++c)
#pragma unroll
    for (int i = 0; i < MT; ++i) {
      acc[c][i] = f32x4_t{0.f, 0.f, 0.f, 0.f};
      if (has_shift) {
#pragma unroll
        for (int f = 0; f < NF; ++f)
          acc[c][i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wf[c][f], sh[i][f], acc[c][i], 0, 0, 0);
      }
    }
  if (norm) {
    // r[m] from the per-tile row sums: thread (part, row) adds tiles part, part + 4, ...
    float ssum = 0.f;
#pragma unroll
    for (int j = 0; j < 16; ++j) ssum += sq[j];
    sm.rowsq[row][part] = ssum;
    __syncthreads();
    if (tid < 64) {
      const float t = (sm.rowsq[tid][0] + sm.rowsq[tid][1]) + (sm.rowsq[tid][2] + sm.rowsq[tid][3]);
      const float ms = t / (float)g.K + g.eps;
      sm.rscale[tid] = 1.0f / sqrtf(ms);
      sm.rowsq[tid][16] = sqrtf(ms);
    }
    __syncthreads();
    if (has_shift) {
#pragma unroll
      for (int i = 0; i < MT; ++i) {
        const float rms = sm.rowsq[i * 16 + l16][16];
#pragma unroll
        for (int c = 0; c < 4; ++c)
#pragma unroll
          for (int q = 0; q < 4; ++q) acc[c][i][q] *= rms;
      }
    }
  }
#pragma unroll
  for (int c = 0; c < 4; ++c)
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
      for (int f = 0; f < NF; ++f)
        acc[c][i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wf[c][f], af[i][f], acc[c][i], 0, 0, 0);
  if (norm) {
#pragma unroll
    for (int i = 0; i < MT; ++i) {
      const float r = sm.rscale[i * 16 + l16];
#pragma unroll
      for (int c = 0; c < 4; ++c)
#pragma unroll
        for (int q = 0; q < 4; ++q) acc[c][i][q] *= r;
    }
  }
  // reduce the four K quarters through LDS.  Item it = tid + 256 q (q < MT) is
  // fragment fr = it >> 6 (= c * MT + i), lane ln = it & 63: row i*16 + (ln & 15),
  // columns n0 + 16c + 4(ln >> 4) .. +3.
  __syncthreads();
#pragma unroll
  for (int c = 0; c < 4; ++c)
#pragma unroll
    for (int i = 0; i < MT; ++i) *(f32x4_t*)&sm.red[wave][c * MT + i][lane][0] = acc[c][i];
  __syncthreads();
  f32x4_t sum[MT];
#pragma unroll
  for (int q = 0; q < MT; ++q) {
    const int it = tid + q * 256;
    sum[q] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const f32x4_t v = *(const f32x4_t*)&sm.red[w][it >> 6][it & 63][0];
      sum[q][0] += v[0];
      sum[q][1] += v[1];
      sum[q][2] += v[2];
      sum[q][3] += v[3];
    }
  }
  auto row_of = [&](int q) { return ((tid + q * 256) >> 6) % MT * 16 + ((tid + q * 256) & 15); };
  auto col_of = [&](int q) { return n0 + ((tid + q * 256) >> 6) / MT * 16 + (((tid + q * 256) & 63) >> 4) * 4; };

  const bool resid = g.e_mode == PE_RESID;
  // epilogue operands (residual x, gate, next-norm scale, bias), one batch
  f32x4_t e_x[MT], e_g[MT], e_s[MT], e_b[MT];
  auto load_epilogue = [&]() {
    const rsrc_t rX = rsrc(g.x_in), rG = rsrc(g.gate), rN = rsrc(g.ns), rB = rsrc(g.bias);
#pragma unroll
    for (int q = 0; q < MT; ++q) {
      const int m = row_of(q), n = col_of(q);
      const bool ok = m < g.M && n + 4 <= g.N;
      e_x[q] = ld_f4<PLAIN>(rX, boff(resid && ok, ((size_t)m * g.ldof + n) * 4));
      e_g[q] = ld_f4<PLAIN>(rG, boff(resid && ok && g.gate, ((size_t)m * g.ldg + n) * 4));
      e_s[q] = ld_f4<PLAIN>(rN, boff(resid && ok, (g.ns_mode == NS_ROW ? (size_t)m * g.ldns + n : (size_t)n) * 4));
      e_b[q] = ld_f4<PLAIN>(rB, boff(!resid && ok && g.bias, (size_t)n * 4));
    }
  };
  if (g.ksplit > 1) {
    // split partial tiles [z][tile] are row-major [MT * 16 rows][64 columns] fp32
    const size_t tile_elems = (size_t)MT * 4 * 64 * 4;
    const rsrc_t rPw = rsrc(g.partial);
#pragma unroll
    for (int q = 0; q < MT; ++q)
      if (row_of(q) < g.M)
        st_f4(rPw, (((size_t)z * tiles + tile) * tile_elems + (size_t)row_of(q) * 64 + (col_of(q) - n0)) * 4, sum[q]);
    if (g.coop) {
      unsigned* ctr = &g.counters[tile * kCounterStride];
      if (group_meet(ctr, (unsigned)g.ksplit, err, &sm.flag)) coop_epilogue<MT>(g, tile, z, tiles, sm, ops);
      __syncthreads();
      return;
    }
    if (!last_arrival(&g.counters[tile * kCounterStride], (unsigned)g.ksplit, &sm.flag)) {
      __syncthreads();
      return;
    }
    // the other K ranges, all in flight at once (with the epilogue operands),
    // added in fixed order
    load_epilogue();
    const rsrc_t rP = rsrc(g.partial);
    f32x4_t pv[MT][kMaxKSplit];
#pragma unroll
    for (int q = 0; q < MT; ++q)
#pragma unroll
      for (int zz = 0; zz < kMaxKSplit; ++zz)
        pv[q][zz] = ld_f4<COH>(rP, boff(zz < g.ksplit && zz != z && row_of(q) < g.M,
                                        (((size_t)zz * tiles + tile) * tile_elems + (size_t)row_of(q) * 64 +
                                         (col_of(q) - n0)) * 4));
#pragma unroll
    for (int q = 0; q < MT; ++q) {
      f32x4_t t = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int zz = 0; zz < kMaxKSplit; ++zz) {
        if (zz >= g.ksplit) break;
        const f32x4_t v = (zz == z) ? sum[q] : pv[q][zz];
        t[0] += v[0];
        t[1] += v[1];
        t[2] += v[2];
        t[3] += v[3];
      }
      sum[q] = t;
    }
  }

  if (g.e_mode == PE_GEGLU) {
    // gate fragments are the even 16-column blocks, up the odd ones
    __syncthreads();
#pragma unroll
    for (int q = 0; q < MT; ++q) *(f32x4_t*)&sm.red[0][(tid + q * 256) >> 6][(tid + q * 256) & 63][0] = sum[q];
    __syncthreads();
#pragma unroll
    for (int q = 0; q < MT; ++q) {
      const int it = tid + q * 256, fr = it >> 6, ln = it & 63;
      const int c = fr / MT, i = fr % MT;
      if (c & 1) continue;
      const int m = i * 16 + (ln & 15), ng = n0 + c * 16;
      if (m >= g.M || ng >= g.N) continue;
      const f32x4_t u = *(const f32x4_t*)&sm.red[0][(c + 1) * MT + i][ln][0];
      const f32x4_t gt = sum[q];
      st_bf16x4(rsrc(g.out_t), geglu_off(g, m, (ng >> 5) * 16 + (ln >> 4) * 4), gelu_tanh_f(gt[0]) * u[0],
                gelu_tanh_f(gt[1]) * u[1], gelu_tanh_f(gt[2]) * u[2], gelu_tanh_f(gt[3]) * u[3]);
    }
    __syncthreads();
    return;
  }

  if (g.ksplit == 1) load_epilogue();
  float gsc = 1.f;
  if (resid && !g.gate) gsc = tanhf(*gptr(g.gate_scalar));

#pragma unroll
  for (int q = 0; q < MT; ++q) {
    const int it = tid + q * 256, fr = it >> 6, ln = it & 63;
    const int c = fr / MT, i = fr % MT;
    const int m = row_of(q), n = col_of(q);
    const f32x4_t v = sum[q];
    float sq = 0.f;
    if (m < g.M && n < g.N) {
      if (g.e_mode == PE_BF16) {
        st_bf16x4(rsrc(g.out_t), ((size_t)m * g.ldo + n) * 2, v[0], v[1], v[2], v[3]);
      } else if (g.e_mode == PE_F32) {
        if (n + 4 <= g.N) {
          st_f4(rsrc(g.out_f), ((size_t)m * g.ldof + n) * 4,
                f32x4_t{v[0] + e_b[q][0], v[1] + e_b[q][1], v[2] + e_b[q][2], v[3] + e_b[q][3]});
        } else {
          for (int r = 0; n + r < g.N; ++r)
            st_f1(rsrc(g.out_f), ((size_t)m * g.ldof + n + r) * 4, v[r] + (g.bias ? *gptr(g.bias + n + r) : 0.f));
        }
      } else {  // PE_RESID
        const f32x4_t gt = g.gate ? e_g[q] : f32x4_t{gsc, gsc, gsc, gsc};
        f32x4_t xn;
        xn[0] = e_x[q][0] + gt[0] * v[0];
        xn[1] = e_x[q][1] + gt[1] * v[1];
        xn[2] = e_x[q][2] + gt[2] * v[2];
        xn[3] = e_x[q][3] + gt[3] * v[3];
        st_f4(rsrc(g.out_f), ((size_t)m * g.ldof + n) * 4, xn);
        st_bf16x4(rsrc(g.p_out), p_off(g, m, n), (1.f + e_s[q][0]) * xn[0], (1.f + e_s[q][1]) * xn[1],
                  (1.f + e_s[q][2]) * xn[2], (1.f + e_s[q][3]) * xn[3]);
        sq = xn[0] * xn[0] + xn[1] * xn[1] + xn[2] * xn[2] + xn[3] * xn[3];
      }
    }
    if (resid) sm.rowsq[i * 16 + (ln & 15)][c * 4 + (ln >> 4)] = sq;
  }
  if (resid) {
    // row sums of squares of the tile's 64 new columns, fixed order
    __syncthreads();
    if (tid < MT * 16 && tid < g.M) {
      float s = 0.f;
#pragma unroll
      for (int h = 0; h < 16; ++h) s += sm.rowsq[tid][h];
      st_f1(rsrc(g.sumsq_out), (size_t)(tile * 64 + tid) * g.sq_out_ld * 4, s);
    }
  }
  __syncthreads();
}

// Stages a whole-K item's shift fragments (the same for every item of the phase) in
// LDS with direct-to-LDS buffer loads: fragment (i, f) of wave w -- rows i*16 + (lane
// & 15), K range w K/4 + 32f + 8(lane >> 4) .. +7, 32-column tiles -- lands at
// shs[w][i * 8 + f][lane].  The shift rows were written before the launch, so this is
// issued with the phase's weight prefetch, before the barrier wait.  The compiler
// does not track these loads' writes to LDS: the reader waits for every load of the
// wave (wait_memory) before it reads them.
template <int MT>
RAVEL_DEV void stage_shift(const PGemm& g, PSmem& sm) {
  typedef __attribute__((address_space(3))) void lds_void_t;
  const int tid = local_tid(), lane = tid & 63, wave = tid >> 6, l16 = lane & 15, grp = lane >> 4;
  const int kq = g.K >> 2, kb = wave * kq;
  const rsrc_t rS = rsrc(g.shift);
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int f = 0; f < 8; ++f) {
      const int m = i * 16 + l16, k = kb + f * 32 + grp * 8;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rS, (lds_void_t*)&sm.shs[wave][i * 8 + f][0], 16,
                                               boff(m < g.M && f * 32 < kq, t32_off(m, k)), 0, 0, 0);
    }
}

// A whole-K item: 16 * WK output columns of every row over the whole K, so the
// item owns its outputs and no other block meets it.  The four waves take K
// quarters of the item (all their loads -- shift rows, activations, row sums --
// issued as one batch), are added through LDS in wave order, and thread
// (i, lane) of the first MT * 64 writes row i*16 + (lane & 15), columns
// n0 + 16c + 4(lane >> 4) .. +3 of every block c: bf16, fp32 plus bias, or
// gelu(gate) * up of the block pair (gate block c = 0, up block c = 1).  The
// norm's operand h = r p + shift is applied as in the split item.  Outputs
// are narrower than a 128-byte line, so the phases that read them use
// device-coherent loads.
template <int MT, int WK>
RAVEL_DEV void gemm_item_wk(const PGemm& g, int item, const u32x4_t (&w16)[16], PSmem& sm, bool sh_staged) {
  bf16x8_t wf[WK][8];
#pragma unroll
  for (int c = 0; c < WK; ++c)
#pragma unroll
    for (int f = 0; f < 8; ++f) wf[c][f] = __builtin_bit_cast(bf16x8_t, w16[c * 8 + f]);
  const int tid = local_tid(), lane = tid & 63, wave = tid >> 6;
  const int l16 = lane & 15, grp = lane >> 4;
  const int n0 = item * 16 * WK, kq = g.K >> 2, kb = wave * kq;
  const bool norm = g.a_mode == PA_NORM;
  const bool has_shift = norm && g.shift != nullptr;
  const rsrc_t rA = rsrc(g.A);
  // The shift fragments go to LDS (staged with the weight prefetch for the block's
  // first item), the activation fragments to registers; every load of the item is
  // in flight at once, and the MFMAs start when all have landed.
  if (has_shift && !sh_staged) stage_shift<MT>(g, sm);
  bf16x8_t x[MT][8];
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int f = 0; f < 8; ++f) {
      const int m = i * 16 + l16, k = kb + f * 32 + grp * 8;
      x[i][f] = ld_b8<PLAIN>(rA, boff(m < g.M && f * 32 < kq, t32_off(m, k)));
    }
  float sq[16];
  const int row = tid & 63, part = tid >> 6, nt = g.K >> 6;
  {
    const rsrc_t rQ = rsrc(g.sumsq_in);
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      const int t = part + 4 * j;
      sq[j] = ld_f1<PLAIN>(rQ, boff(norm && t < nt && row < g.M, (size_t)(t * 64 + row) * g.sq_in_ld * 4));
    }
  }
  f32x4_t bias4 = {0.f, 0.f, 0.f, 0.f};
  {
    const int n = n0 + 4 * ((tid & 63) >> 4);
    bias4 = ld_f4<PLAIN>(rsrc(g.bias), boff(g.e_mode == PE_F32 && g.bias && n + 4 <= g.N, (size_t)n * 4));
  }
  wait_memory();  // includes the direct-to-LDS shift loads

  f32x4_t acc[WK][MT];
#pragma unroll
  for (int c = 0; c < WK; ++c)
#pragma unroll
    for (int i = 0; i < MT; ++i) acc[c][i] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  if (has_shift) {
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
      for (int f = 0; f < 8; ++f) {
        const bf16x8_t s = __builtin_bit_cast(bf16x8_t, sm.shs[wave][i * 8 + f][lane]);
#pragma unroll
        for (int c = 0; c < WK; ++c) acc[c][i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wf[c][f], s, acc[c][i], 0, 0, 0);
      }
  }
  if (norm) {
    float ssum = 0.f;
#pragma unroll
    for (int j = 0; j < 16; ++j) ssum += sq[j];
    sm.rowsq[row][part] = ssum;
    __syncthreads();
    if (tid < 64) {
      const float t = (sm.rowsq[tid][0] + sm.rowsq[tid][1]) + (sm.rowsq[tid][2] + sm.rowsq[tid][3]);
      const float ms = t / (float)g.K + g.eps;
      sm.rscale[tid] = 1.0f / sqrtf(ms);
      sm.rowsq[tid][16] = sqrtf(ms);
    }
    __syncthreads();
    if (has_shift) {
#pragma unroll
      for (int i = 0; i < MT; ++i) {
        const float rms = sm.rowsq[i * 16 + l16][16];
#pragma unroll
        for (int c = 0; c < WK; ++c)
#pragma unroll
          for (int q = 0; q < 4; ++q) acc[c][i][q] *= rms;
      }
    }
  }
#pragma unroll
  for (int c = 0; c < WK; ++c)
#pragma unroll
    for (int i = 0; i < MT; ++i)
#pragma unroll
      for (int f = 0; f < 8; ++f)
        acc[c][i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wf[c][f], x[i][f], acc[c][i], 0, 0, 0);
  if (norm) {
#pragma unroll
    for (int i = 0; i < MT; ++i) {
      const float r = sm.rscale[i * 16 + l16];
#pragma unroll
      for (int c = 0; c < WK; ++c)
#pragma unroll
        for (int q = 0; q < 4; ++q) acc[c][i][q] *= r;
    }
  }
  __syncthreads();
#pragma unroll
  for (int c = 0; c < WK; ++c)
#pragma unroll
    for (int i = 0; i < MT; ++i) *(f32x4_t*)&sm.red[wave][c * MT + i][lane][0] = acc[c][i];
  __syncthreads();
  if (tid < MT * 64) {
    const int i = tid >> 6, ln = tid & 63;
    const int m = i * 16 + (ln & 15), cg = 4 * (ln >> 4);
    f32x4_t s[WK];
#pragma unroll
    for (int c = 0; c < WK; ++c) {
      s[c] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        const f32x4_t v = *(const f32x4_t*)&sm.red[w][c * MT + i][ln][0];
        s[c][0] += v[0];
        s[c][1] += v[1];
        s[c][2] += v[2];
        s[c][3] += v[3];
      }
    }
    if (m < g.M) {
      if constexpr (WK == 2) {
        if (g.e_mode == PE_GEGLU) {
          st_bf16x4(rsrc(g.out_t), geglu_off(g, m, item * 16 + cg), gelu_tanh_f(s[0][0]) * s[1][0],
                    gelu_tanh_f(s[0][1]) * s[1][1], gelu_tanh_f(s[0][2]) * s[1][2], gelu_tanh_f(s[0][3]) * s[1][3]);
        }
      }
      if (g.e_mode == PE_BF16) {
#pragma unroll
        for (int c = 0; c < WK; ++c) {
          const int n = n0 + 16 * c + cg;
          if (n < g.N) st_bf16x4(rsrc(g.out_t), ((size_t)m * g.ldo + n) * 2, s[c][0], s[c][1], s[c][2], s[c][3]);
        }
      } else if (g.e_mode == PE_F32) {
        const int n = n0 + cg;  // PE_F32 items have one column block
        if (n + 4 <= g.N) {
          st_f4(rsrc(g.out_f), ((size_t)m * g.ldof + n) * 4,
                f32x4_t{s[0][0] + bias4[0], s[0][1] + bias4[1], s[0][2] + bias4[2], s[0][3] + bias4[3]});
        } else {
          for (int r = 0; n + r < g.N; ++r)
            st_f1(rsrc(g.out_f), ((size_t)m * g.ldof + n + r) * 4, s[0][r] + (g.bias ? *gptr(g.bias + n + r) : 0.f));
        }
      }
    }
  }
  __syncthreads();
}

// One item of a phase's side work (PSide): 32 output columns n0 .. n0 + 31 of every
// row over the whole K, the four waves taking K quarters (K/4 a multiple of 32, at
// most 256) added in LDS; run by a block with no item of its own in the phase, off
// the phase's critical path.
template <int MT>
RAVEL_DEV void side_item(const PSide& sd, int item, PSmem& sm) {
  const int tid = local_tid(), lane = tid & 63, wave = tid >> 6;
  const int l16 = lane & 15, grp = lane >> 4;
  const int n0 = item * 32, kq = sd.K >> 2, kb = wave * kq;
  const rsrc_t rW = rsrc(sd.W), rA = rsrc(sd.A);
  bf16x8_t wf[2][8], af[MT][8];
#pragma unroll
  for (int c = 0; c < 2; ++c)
#pragma unroll
    for (int f = 0; f < 8; ++f) {
      const int n = n0 + c * 16 + l16, k = kb + f * 32 + grp * 8;
      wf[c][f] = ld_b8<PLAIN>(rW, boff(f * 32 < kq && n < sd.N, ((size_t)n * sd.ldw + k) * 2));
    }
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int f = 0; f < 8; ++f) {
      const int m = i * 16 + l16, k = kb + f * 32 + grp * 8;
      af[i][f] = ld_b8<PLAIN>(rA, boff(f * 32 < kq && m < sd.M, ((size_t)m * sd.lda + k) * 2));
    }
  f32x4_t bias4[2];
#pragma unroll
  for (int c = 0; c < 2; ++c) {
    const int n = n0 + c * 16 + 4 * ((tid & 63) >> 4);
    bias4[c] = ld_f4<PLAIN>(rsrc(sd.bias), boff(n + 4 <= sd.N, (size_t)n * 4));
  }
  f32x4_t acc[2][MT];
#pragma unroll
  for (int c = 0; c < 2; ++c)
#pragma unroll
    for (int i = 0; i < MT; ++i) {
      acc[c][i] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int f = 0; f < 8; ++f) acc[c][i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wf[c][f], af[i][f], acc[c][i], 0, 0, 0);
    }
  __syncthreads();
#pragma unroll
  for (int c = 0; c < 2; ++c)
#pragma unroll
    for (int i = 0; i < MT; ++i) *(f32x4_t*)&sm.red[wave][c * MT + i][lane][0] = acc[c][i];
  __syncthreads();
  if (tid < MT * 64) {
    const int i = tid >> 6, ln = tid & 63;
    const int m = i * 16 + (ln & 15), cg = 4 * (ln >> 4);
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      f32x4_t s = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        const f32x4_t v = *(const f32x4_t*)&sm.red[w][c * MT + i][ln][0];
        s[0] += v[0];
        s[1] += v[1];
        s[2] += v[2];
        s[3] += v[3];
      }
      const int n = n0 + c * 16 + cg;
      if (m < sd.M && n + 4 <= sd.N) {
        const f32x4_t o = {s[0] + bias4[c][0], s[1] + bias4[c][1], s[2] + bias4[c][2], s[3] + bias4[c][3]};
        st_f4(rsrc(sd.out), ((size_t)m * sd.ldo + n) * 4, o);
#pragma unroll
        for (int r = 0; r < 2; ++r) {
          const int col = n - sd.shift_col[r];
          if (sd.shift_out[r] && col >= 0 && col < sd.shift_w)
            st_bf16x4(rsrc(sd.shift_out[r]), t32_off(m, col), o[0], o[1], o[2], o[3]);
        }
      }
    }
  }
  __syncthreads();
}

// A split-K tile finished by its ksplit blocks together: block z takes rows
// [z*rp, min(M, (z+1)*rp)), rp = ceil(M / ksplit), adds the partials of each of its
// (row, 4-column) slots in split order and applies the epilogue; the new rows' sums
// of squares of a residual update are added in fixed column order.
// Slot s of the block's share: row r0 + s / per_row, 4-column group and 16-column
// block (GEGLU: block pair) from s % per_row.
struct CoopSlot {
  int row, grp, cb, c, n;
  bool valid, ok;
};
template <int MT>
RAVEL_DEV CoopSlot coop_slot(const PGemm& g, int tile, int z, int slot) {
  const int rp = coop_rows(g);
  const int r0 = z * rp, r1 = min(g.M, r0 + rp);
  const bool geglu = g.e_mode == PE_GEGLU;
  const int per_row = geglu ? 8 : 16;
  const int nslots = max(r1 - r0, 0) * per_row;
  CoopSlot q;
  q.valid = slot < nslots;
  q.row = r0 + (q.valid ? slot / per_row : 0);
  const int rem = slot % per_row;
  q.grp = rem & 3;
  q.cb = rem >> 2;
  q.c = geglu ? 2 * q.cb : q.cb;
  q.n = tile * 64 + q.c * 16 + q.grp * 4;
  q.ok = q.valid && q.n + 4 <= g.N;
  return q;
}

template <int MT>
RAVEL_DEV CoopOps coop_operands(const PGemm& g, int tile, int z, int s0, bool use) {
  CoopSlot q = coop_slot<MT>(g, tile, z, s0 + local_tid());
  q.ok = q.ok && use;
  const bool geglu = g.e_mode == PE_GEGLU, resid = g.e_mode == PE_RESID;
  const rsrc_t rX = rsrc(g.x_in), rG = rsrc(g.gate), rN = rsrc(g.ns), rB = rsrc(g.bias);
  CoopOps o;
  o.ex = ld_f4<PLAIN>(rX, boff(resid && q.ok, ((size_t)q.row * g.ldof + q.n) * 4));
  o.eg = ld_f4<PLAIN>(rG, boff(resid && q.ok && g.gate, ((size_t)q.row * g.ldg + q.n) * 4));
  o.es = ld_f4<PLAIN>(rN, boff(resid && q.ok, (g.ns_mode == NS_ROW ? (size_t)q.row * g.ldns + q.n : (size_t)q.n) * 4));
  o.eb = ld_f4<PLAIN>(rB, boff(!resid && !geglu && q.ok && g.bias, (size_t)q.n * 4));
  return o;
}

// A split-K tile finished by its ksplit blocks together: block z takes rows
// [z*rp, min(M, (z+1)*rp)), rp = ceil(M / ksplit), adds the partials of each of its
// (row, 4-column) slots in split order and applies the epilogue; the new rows' sums
// of squares of a residual update are added in fixed column order.
template <int MT>
RAVEL_DEV void coop_epilogue(const PGemm& g, int tile, int z, int tiles, PSmem& sm, const CoopOps& first) {
  const int tid = local_tid();
  const int n0 = tile * 64;
  const int rp = coop_rows(g);
  const int r0 = z * rp, r1 = min(g.M, r0 + rp);
  const size_t tile_elems = (size_t)MT * 4 * 64 * 4;
  const bool geglu = g.e_mode == PE_GEGLU, resid = g.e_mode == PE_RESID;
  const int per_row = geglu ? 8 : 16;
  const int nslots = max(r1 - r0, 0) * per_row;
  const rsrc_t rP = rsrc(g.partial);
  float gsc = 1.f;
  if (resid && !g.gate) gsc = tanhf(*gptr(g.gate_scalar));
  for (int s0 = 0; s0 < nslots; s0 += 256) {
    const CoopSlot q = coop_slot<MT>(g, tile, z, s0 + tid);
    const bool valid = q.valid;
    const int row = q.row, grp = q.grp, cb = q.cb, c = q.c, n = q.n;
    const CoopOps o = s0 == 0 ? first : coop_operands<MT>(g, tile, z, s0, true);
    const f32x4_t ex = o.ex, eg = o.eg, es = o.es, eb = o.eb;
    // the slot's 4 columns in the row-major partial tiles (16 consecutive slots read
    // one row), and for GeGLU those of the up block 16 columns on
    const size_t el = (size_t)row * 64 + (n - n0);
    f32x4_t pv[kMaxKSplit], pu[kMaxKSplit];
#pragma unroll
    for (int zz = 0; zz < kMaxKSplit; ++zz)
      pv[zz] = ld_f4<COH>(rP, boff(valid && zz < g.ksplit, (((size_t)zz * tiles + tile) * tile_elems + el) * 4));
#pragma unroll
    for (int zz = 0; zz < kMaxKSplit; ++zz) pu[zz] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    if (geglu) {
#pragma unroll
      for (int zz = 0; zz < kMaxKSplit; ++zz)
        pu[zz] = ld_f4<COH>(rP, boff(valid && zz < g.ksplit, (((size_t)zz * tiles + tile) * tile_elems + el + 16) * 4));
    }
    f32x4_t v = {0.f, 0.f, 0.f, 0.f}, u = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int zz = 0; zz < kMaxKSplit; ++zz) {
      if (zz >= g.ksplit) break;
      v[0] += pv[zz][0];
      v[1] += pv[zz][1];
      v[2] += pv[zz][2];
      v[3] += pv[zz][3];
      u[0] += pu[zz][0];
      u[1] += pu[zz][1];
      u[2] += pu[zz][2];
      u[3] += pu[zz][3];
    }
    float sq = 0.f;
    if (valid && n < g.N) {
      if (geglu) {
        st_bf16x4(rsrc(g.out_t), geglu_off(g, row, (n0 >> 1) + cb * 16 + grp * 4), gelu_tanh_f(v[0]) * u[0],
                  gelu_tanh_f(v[1]) * u[1], gelu_tanh_f(v[2]) * u[2], gelu_tanh_f(v[3]) * u[3]);
      } else if (g.e_mode == PE_BF16) {
        st_bf16x4(rsrc(g.out_t), ((size_t)row * g.ldo + n) * 2, v[0], v[1], v[2], v[3]);
      } else if (g.e_mode == PE_F32) {
        if (n + 4 <= g.N) {
          st_f4(rsrc(g.out_f), ((size_t)row * g.ldof + n) * 4, f32x4_t{v[0] + eb[0], v[1] + eb[1], v[2] + eb[2], v[3] + eb[3]});
        } else {
          for (int r = 0; n + r < g.N; ++r)
            st_f1(rsrc(g.out_f), ((size_t)row * g.ldof + n + r) * 4, v[r] + (g.bias ? *gptr(g.bias + n + r) : 0.f));
        }
      } else {  // PE_RESID
        const f32x4_t gt = g.gate ? eg : f32x4_t{gsc, gsc, gsc, gsc};
        f32x4_t xn;
        xn[0] = ex[0] + gt[0] * v[0];
        xn[1] = ex[1] + gt[1] * v[1];
        xn[2] = ex[2] + gt[2] * v[2];
        xn[3] = ex[3] + gt[3] * v[3];
        st_f4(rsrc(g.out_f), ((size_t)row * g.ldof + n) * 4, xn);
        st_bf16x4(rsrc(g.p_out), p_off(g, row, n), (1.f + es[0]) * xn[0], (1.f + es[1]) * xn[1],
                  (1.f + es[2]) * xn[2], (1.f + es[3]) * xn[3]);
        sq = xn[0] * xn[0] + xn[1] * xn[1] + xn[2] * xn[2] + xn[3] * xn[3];
      }
    }
    if (resid && valid) sm.rowsq[row - r0][c * 4 + grp] = sq;
  }
  if (resid) {
    __syncthreads();
    if (tid < r1 - r0) {
      float s = 0.f;
#pragma unroll
      for (int h = 0; h < 16; ++h) s += sm.rowsq[tid][h];
      st_f1(rsrc(g.sumsq_out), (size_t)(tile * 64 + r0 + tid) * g.sq_out_ld * 4, s);
    }
  }
}

// ---------------------------------------------------------------------------
// attention: one (env, head, key split)
// ---------------------------------------------------------------------------
// Where the keys of item's split start and end, and whether they are prefix keys.
struct SplitKeys {
  int e, j, g, split, kbeg, kend;
  bool self;
};
RAVEL_DEV SplitKeys split_keys(const AttnArgs& a, int item) {
  SplitKeys k;
  k.split = item % a.nsplit;
  k.j = (item / a.nsplit) % a.nq;
  k.e = item / (a.nsplit * a.nq);
  k.g = (k.j * a.nkv) / a.nq;
  // the first ceil(P / kps) splits cover the prefix, the rest the self keys
  const int nsp = (a.P + a.keys_per_split - 1) / a.keys_per_split;
  k.self = k.split >= nsp;
  k.kbeg = k.self ? a.P + (k.split - nsp) * a.keys_per_split : k.split * a.keys_per_split;
  k.kend = k.self ? min(a.P + a.S, k.kbeg + a.keys_per_split) : min(a.P, k.kbeg + a.keys_per_split);
  return k;
}

// The split's keys and values into registers: kv[0..3] are 16-byte K chunks
// (chunk c = tid + 256 r: key c / (HD/8), dims (c % (HD/8)) * 8), kv[4..7] the V
// chunks of keys 4 (tid / (HD/8)) + i, i < 4, at dims (tid % (HD/8)) * 8.  Prefix
// rows were written before the launch (plain loads, and may be fetched before the
// barrier that opens the phase); self rows by this launch (coherent loads).
template <int HD, int AUX>
RAVEL_DEV void attn_load_kv_aux(const AttnArgs& a, const SplitKeys& k, const int* slots, u32x4_t (&kv)[8]) {
  constexpr int CPR = HD / 8;
  const int tid = local_tid();
  const int slot = a.slot ? slots[k.e] : 0;
  const bf16_t* pk = (const bf16_t*)a.pk + slot * a.p_slot_stride + k.e * a.p_env_stride;
  const bf16_t* pv = (const bf16_t*)a.pv + slot * a.p_slot_stride + k.e * a.p_env_stride;
  const rsrc_t rK = k.self ? rsrc((const bf16_t*)a.sk + (size_t)k.e * a.S * a.s_ld) : rsrc(pk);
  const rsrc_t rV = k.self ? rsrc((const bf16_t*)a.sv + (size_t)k.e * a.S * a.s_ld) : rsrc(pv);
  const int ld_row = k.self ? a.s_ld : a.p_ld;
  const int k_row0 = k.self ? a.P : 0;
  auto off = [&](int kidx, int dc) {
    return boff(kidx < k.kend, ((size_t)(kidx - k_row0) * ld_row + k.g * HD + dc) * 2);
  };
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int c = tid + r * 256;
    const int o = off(k.kbeg + c / CPR, (c % CPR) * 8);
    kv[r] = ld16<AUX>(rK, o);
  }
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int o = off(k.kbeg + (tid / CPR) * 4 + i, (tid % CPR) * 8);
    kv[4 + i] = ld16<AUX>(rV, o);
  }
}
// Self rows written in 16-column pieces (a.coh) are read device-coherent.
template <int HD>
RAVEL_DEV void attn_load_kv(const AttnArgs& a, const SplitKeys& k, const int* slots, u32x4_t (&kv)[8]) {
  if (k.self && a.coh)
    attn_load_kv_aux<HD, COH>(a, k, slots, kv);
  else
    attn_load_kv_aux<HD, PLAIN>(a, k, slots, kv);
}

// Weighted sum of the splits' partial outputs for output elements [el0, el1) of
// one (env, head) (element = 4 dims of one query), bf16 to a.out.  Split s holds its
// output normalised by its own sum l_s (fp16) and its maximum m_s; its weight for
// query q is exp2(m_s - m) l_s / sum_s' exp2(m_s' - m) l_s' (fixed order).
template <int HD>
RAVEL_DEV void attn_merge(const AttnArgs& a, int e, int j, int el0, int el1, PSmem& sm) {
  const int tid = local_tid();
  const int Hp = ((a.Hq + 15) / 16) * 16;
  const size_t pbase = ((size_t)e * a.nq + j) * a.nsplit;
  const rsrc_t rML = rsrc(a.part_ml), rO = rsrc(a.part_o);
  // (max, sum) of every split and query: kMaxAttnSplit x 64 pairs, 8 per thread
  float2 mlv[8];
#pragma unroll
  for (int r = 0; r < 8; ++r) {
    const int t = tid + r * 256, sp = t >> 6, qq = t & 63;
    mlv[r] = ld_f2<COH>(rML, boff(sp < a.nsplit && qq < a.Hq, ((pbase + sp) * Hp + qq) * 2 * 4));
  }
  // each thread sums one element over the splits, 16 splits per batch of loads
  constexpr int SB = 16;
  f32x4_t pvl[SB];
  auto load_parts = [&](int el, int sp0) {
    const int qq = el / (HD / 4), d = (el % (HD / 4)) * 4;
#pragma unroll
    for (int i = 0; i < SB; ++i)
      pvl[i] = ld_f16x4<COH>(rO, boff(el < el1 && sp0 + i < a.nsplit, (((pbase + sp0 + i) * Hp + qq) * HD + d) * 2));
  };
  load_parts(el0 + tid, 0);  // in flight with the (max, sum) loads
#pragma unroll
  for (int r = 0; r < 8; ++r) {
    const int t = tid + r * 256, sp = t >> 6, qq = t & 63;
    sm.mg.ml[sp][qq][0] = (sp < a.nsplit && qq < a.Hq) ? mlv[r].x : -INFINITY;
    sm.mg.ml[sp][qq][1] = mlv[r].y;
  }
  __syncthreads();
  if (tid < a.Hq) {
    float mmax = -INFINITY;
    for (int sp = 0; sp < a.nsplit; ++sp) mmax = fmaxf(mmax, sm.mg.ml[sp][tid][0]);
    float den = 0.f;
    for (int sp = 0; sp < a.nsplit; ++sp) {
      const float ms = sm.mg.ml[sp][tid][0];
      const float wv = (ms == -INFINITY) ? 0.f : exp2f(ms - mmax);
      sm.mg.wgt[sp][tid] = wv * sm.mg.ml[sp][tid][1];
      den += wv * sm.mg.ml[sp][tid][1];
    }
    const float inv = 1.f / den;
    for (int sp = 0; sp < a.nsplit; ++sp) sm.mg.wgt[sp][tid] *= inv;
  }
  __syncthreads();
  for (int b0 = el0; b0 < el1; b0 += 256) {
    const int el = b0 + tid;
    const int qq = el < el1 ? el / (HD / 4) : 0, d = (el % (HD / 4)) * 4;
    f32x4_t num = {0.f, 0.f, 0.f, 0.f};
    for (int sp0 = 0; sp0 < a.nsplit; sp0 += SB) {
      if (b0 != el0 || sp0 != 0) load_parts(el, sp0);
#pragma unroll
      for (int i = 0; i < SB; ++i) {
        if (sp0 + i >= a.nsplit) break;
        const float wv = sm.mg.wgt[sp0 + i][qq];
        num[0] += wv * pvl[i][0];
        num[1] += wv * pvl[i][1];
        num[2] += wv * pvl[i][2];
        num[3] += wv * pvl[i][3];
      }
    }
    if (el < el1)
      st_bf16x4(rsrc(a.out), ((size_t)(e * a.Hq + qq) * a.ldo + j * HD + d) * 2, num[0], num[1], num[2], num[3]);
  }
}

// The same merge in one round of loads, for a share of at most 128 elements and at
// most kMaxAttnSplit splits: thread (h, j) = (tid / 128, tid % 128) takes element
// el0 + j and the splits of parity h; it loads the (max, sum) of every split of
// its query (one address per wave: the wave's elements share a query when HD >= 256,
// a few queries otherwise) and its 16 partial outputs together, forms the weights
// in registers, and the two halves are added through LDS (even splits, then odd).
template <int HD>
RAVEL_DEV void attn_merge_one_round(const AttnArgs& a, int e, int j, int el0, int el1, PSmem& sm) {
  const int tid = local_tid(), h = tid >> 7, el = el0 + (tid & 127);
  const int Hp = ((a.Hq + 15) / 16) * 16;
  const size_t pbase = ((size_t)e * a.nq + j) * a.nsplit;
  const rsrc_t rML = rsrc(a.part_ml), rO = rsrc(a.part_o);
  const bool valid = el < el1;
  const int qq = valid ? el / (HD / 4) : 0, d = (el % (HD / 4)) * 4;
  f32x4_t pv[kMaxAttnSplit / 2];
  if constexpr (HD == 256) {
    // a wave's 64 elements are one query (shares start at multiples of 64 elements):
    // lane s loads split s's (max, sum), the weights are reduced across the wave, and
    // each thread takes the weights of its splits from their lanes
    const int lane = tid & 63, e0 = el0 + (tid & 64);
    const int qw = e0 / 64;
    const float2 mls = ld_f2<COH>(rML, boff(e0 < el1 && lane < a.nsplit, ((pbase + lane) * Hp + qw) * 2 * 4));
#pragma unroll
    for (int i = 0; i < kMaxAttnSplit / 2; ++i) {
      const int sp = 2 * i + h;
      pv[i] = ld_f16x4<COH>(rO, boff(valid && sp < a.nsplit, (((pbase + sp) * Hp + qq) * HD + d) * 2));
    }
    const bool use = lane < a.nsplit && mls.x != -INFINITY;
    float mmax = use ? mls.x : -INFINITY;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) mmax = fmaxf(mmax, __shfl_xor(mmax, o, 64));
    const float ws = use ? exp2f(mls.x - mmax) * mls.y : 0.f;
    float den = ws;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) den += __shfl_xor(den, o, 64);
    f32x4_t num = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int i = 0; i < kMaxAttnSplit / 2; ++i) {
      const float w = __shfl(ws, 2 * i + h, 64);
      num[0] += w * pv[i][0];
      num[1] += w * pv[i][1];
      num[2] += w * pv[i][2];
      num[3] += w * pv[i][3];
    }
    f32x4_t* x = reinterpret_cast<f32x4_t*>(&sm.red[0][0][0][0]);
    if (h == 1) x[tid & 127] = num;
    __syncthreads();
    if (h == 0 && valid) {
      const f32x4_t o = x[tid];
      const float inv = 1.f / den;
      st_bf16x4(rsrc(a.out), ((size_t)(e * a.Hq + qq) * a.ldo + j * HD + d) * 2, (num[0] + o[0]) * inv,
                (num[1] + o[1]) * inv, (num[2] + o[2]) * inv, (num[3] + o[3]) * inv);
    }
    return;
  }
  float2 ml[kMaxAttnSplit];
#pragma unroll
  for (int sp = 0; sp < kMaxAttnSplit; ++sp)
    ml[sp] = ld_f2<COH>(rML, boff(valid && sp < a.nsplit, ((pbase + sp) * Hp + qq) * 2 * 4));
#pragma unroll
  for (int i = 0; i < kMaxAttnSplit / 2; ++i) {
    const int sp = 2 * i + h;
    pv[i] = ld_f16x4<COH>(rO, boff(valid && sp < a.nsplit, (((pbase + sp) * Hp + qq) * HD + d) * 2));
  }
  // splits past nsplit read (0, 0): they are masked out of the max and get weight 0
  float mmax = -INFINITY;
#pragma unroll
  for (int sp = 0; sp < kMaxAttnSplit; ++sp) mmax = fmaxf(mmax, sp < a.nsplit ? ml[sp].x : -INFINITY);
  float den = 0.f;
  f32x4_t num = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int sp = 0; sp < kMaxAttnSplit; ++sp) {
    const bool use = sp < a.nsplit && ml[sp].x != -INFINITY;
    const float wv = use ? exp2f(ml[sp].x - mmax) * ml[sp].y : 0.f;
    den += wv;
    const float wh = (sp & 1) == h ? wv : 0.f;
    const f32x4_t p = pv[sp >> 1];
    num[0] += wh * p[0];
    num[1] += wh * p[1];
    num[2] += wh * p[2];
    num[3] += wh * p[3];
  }
  f32x4_t* x = reinterpret_cast<f32x4_t*>(&sm.red[0][0][0][0]);
  if (h == 1) x[tid & 127] = num;
  __syncthreads();
  if (h == 0 && valid) {
    const f32x4_t o = x[tid];
    const float inv = 1.f / den;
    st_bf16x4(rsrc(a.out), ((size_t)(e * a.Hq + qq) * a.ldo + j * HD + d) * 2, (num[0] + o[0]) * inv,
              (num[1] + o[1]) * inv, (num[2] + o[2]) * inv, (num[3] + o[3]) * inv);
  }
}

// One split: its keys and values (kv, fetched ahead when `have_kv`) are staged in
// LDS, the four waves take 16 queries each, S^T = K Q^T with the split's softmax,
// O^T = V^T P^T; a single split writes the output, otherwise the splits' partial
// outputs and (max, sum) are merged by the head's splits together (coop) or by the
// last split to arrive.
template <int HD, class AfterLoads>
RAVEL_DEV void attn_item(const AttnArgs& a, int item, const int* slots, int* err, PSmem& sm, u32x4_t (&kv)[8],
                         bool have_kv, AfterLoads&& after_loads) {
  using C = AttnCfg<HD>;
  constexpr int KPS = C::KPS, KLD = C::KLD, VLD = C::VLD;
  constexpr int KS = HD / 32, DT = HD / 16, CPR = HD / 8;
  bf16_t* Ks = sm.at;
  bf16_t* Vt = sm.at + KPS * KLD;
  const int tid = local_tid(), lane = tid & 63, wave = tid >> 6;
  const int l16 = lane & 15, grp = lane >> 4;
  const SplitKeys k = split_keys(a, item);
  const int e = k.e, j = k.j, split = k.split;
  const int QB = (a.Hq + 15) / 16;
  if (!have_kv) attn_load_kv<HD>(a, k, slots, kv);
  const rsrc_t rq = rsrc(a.q);
  const int query = wave * 16 + l16;
  const bool active = wave < QB;
  bf16x8_t qf[KS];
  auto q_off = [&](int ks) {
    return boff(query < a.Hq, ((size_t)(e * a.Hq + query) * a.ldq + j * HD + ks * 32 + grp * 8) * 2);
  };
  if (a.coh) {
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) qf[ks] = ld_b8<COH>(rq, q_off(ks));
  } else {
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) qf[ks] = ld_b8<PLAIN>(rq, q_off(ks));
  }
  after_loads();
  __syncthreads();  // LDS may still be read by this block's previous item
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    const int c = tid + r * 256;
    *(u32x4_t*)&Ks[(c / CPR) * KLD + (c % CPR) * 8] = kv[r];
  }
  {
    const int kq = tid / CPR, dc = (tid % CPR) * 8;
    const bf16_t* h0 = (const bf16_t*)&kv[4];
    const bf16_t* h1 = (const bf16_t*)&kv[5];
    const bf16_t* h2 = (const bf16_t*)&kv[6];
    const bf16_t* h3 = (const bf16_t*)&kv[7];
#pragma unroll
    for (int dd = 0; dd < 8; ++dd) {
      u32x2_t w;
      w[0] = (uint32_t)h0[dd] | ((uint32_t)h1[dd] << 16);
      w[1] = (uint32_t)h2[dd] | ((uint32_t)h3[dd] << 16);
      *(u32x2_t*)&Vt[(dc + dd) * VLD + kq * 4] = w;
    }
  }
  __syncthreads();

  // A split holds at most KPS keys, so its scores are computed at once: S^T = K Q^T
  // for every 32-key tile t (lane: query l16, keys 32t + 4grp..+3 and 32t + 16 +
  // 4grp..+3) as 2 x NT independent MFMA chains, then one softmax over the split
  // and O^T = V^T P^T with no running rescale.
  constexpr int NT = KPS / 32;
  const int nk = k.kend - k.kbeg;
  const int ntile = (nk + 31) / 32;
  f32x4_t o[DT];
  float mrow = -INFINITY, lrow = 0.f;
#pragma unroll
  for (int dt = 0; dt < DT; ++dt) o[dt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  const float sl2 = a.scale * 1.4426950408889634f;
  if (active) {
    f32x4_t sc[NT][2];
#pragma unroll
    for (int t = 0; t < NT; ++t) sc[t][0] = sc[t][1] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        if (t >= ntile) continue;  // wave-uniform
#pragma unroll
        for (int st = 0; st < 2; ++st) {
          const bf16x8_t kf = *(const bf16x8_t*)&Ks[(t * 32 + st * 16 + l16) * KLD + ks * 32 + grp * 8];
          sc[t][st] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf, qf[ks], sc[t][st], 0, 0, 0);
        }
      }
    float mx = -INFINITY;
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int st = 0; st < 2; ++st)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          float x = sc[t][st][r] * sl2;
          if (t * 32 + st * 16 + grp * 4 + r >= nk) x = -INFINITY;
          sc[t][st][r] = x;
          mx = fmaxf(mx, x);
        }
    mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
    float psum = 0.f;
    bf16x8_t pf[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      float p[2][4];
#pragma unroll
      for (int st = 0; st < 2; ++st)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          p[st][r] = (sc[t][st][r] == -INFINITY) ? 0.f : exp2f(sc[t][st][r] - mx);
          psum += p[st][r];
        }
      const u32x4_t pb = {pack_bf16x2(p[0][0], p[0][1]), pack_bf16x2(p[0][2], p[0][3]), pack_bf16x2(p[1][0], p[1][1]),
                          pack_bf16x2(p[1][2], p[1][3])};
      pf[t] = *reinterpret_cast<const bf16x8_t*>(&pb);
    }
    psum += __shfl_xor(psum, 16, 64);
    psum += __shfl_xor(psum, 32, 64);
    mrow = mx;
    lrow = psum;
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      if (t >= ntile) continue;  // wave-uniform
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        const bf16_t* vrow = &Vt[(dt * 16 + l16) * VLD + t * 32];
        const u32x2_t lo = *(const u32x2_t*)(vrow + grp * 4);
        const u32x2_t hi = *(const u32x2_t*)(vrow + 16 + grp * 4);
        const u32x4_t vv = {lo[0], lo[1], hi[0], hi[1]};
        o[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(*(const bf16x8_t*)&vv, pf[t], o[dt], 0, 0, 0);
      }
    }
  }
  bf16_t* out = (bf16_t*)a.out;
  if (a.nsplit == 1) {
    if (active && query < a.Hq) {
      const float inv = 1.f / lrow;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt)
        st_bf16x4(rsrc(out), ((size_t)(e * a.Hq + query) * a.ldo + j * HD + dt * 16 + grp * 4) * 2, o[dt][0] * inv,
                  o[dt][1] * inv, o[dt][2] * inv, o[dt][3] * inv);
    }
    __syncthreads();
    return;
  }
  const int Hp = QB * 16;
  const size_t pbase = ((size_t)e * a.nq + j) * a.nsplit;
  if (active && query < a.Hq) {
    const rsrc_t rPo = rsrc(a.part_o), rPml = rsrc(a.part_ml);
    const size_t po = ((pbase + split) * Hp + query) * HD;
    // the split's output normalised by its own softmax sum (|values| <= max |v|), fp16
    const float inv = 1.f / lrow;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt)
      st_f16x4(rPo, (po + dt * 16 + grp * 4) * 2,
               f32x4_t{o[dt][0] * inv, o[dt][1] * inv, o[dt][2] * inv, o[dt][3] * inv});
    if (grp == 0) {
      st_f1(rPml, (((pbase + split) * Hp + query) * 2 + 0) * 4, mrow);
      st_f1(rPml, (((pbase + split) * Hp + query) * 2 + 1) * 4, lrow);
    }
  }
  const int total = a.Hq * (HD / 4);
  unsigned* ctr = &a.counters[(e * a.nq + j) * kCounterStride];
  if (a.coop) {
    // the splits of this (env, head) meet; each merges a share of the output
    if (group_meet(ctr, (unsigned)a.nsplit, err, &sm.flag)) {
      // shares of whole 128-byte lines of the bf16 output (16 elements of 4 dims)
      const int share = (((total + a.nsplit - 1) / a.nsplit) + 15) & ~15;
      const int el0 = split * share, el1 = min(total, el0 + share);
      if (share <= 128)
        attn_merge_one_round<HD>(a, e, j, el0, el1, sm);
      else
        attn_merge<HD>(a, e, j, el0, el1, sm);
    }
    __syncthreads();
    return;
  }
  if (last_arrival(ctr, (unsigned)a.nsplit, &sm.flag)) attn_merge<HD>(a, e, j, 0, total, sm);
  __syncthreads();
}

// ---------------------------------------------------------------------------
// the persistent kernel
// ---------------------------------------------------------------------------
constexpr int kDescChunks = (int)(sizeof(Phase) / 16);
static_assert(sizeof(Phase) % 16 == 0 && kDescChunks <= 256, "phase descriptor size");

// One row of a rotary phase: each thread turns four consecutive pairs of one head
// (8-byte loads and stores of the bf16 halves, the loads device-coherent when the
// rows were written in pieces narrower than a line; the angle table was written
// before the launch).
RAVEL_DEV void rope_item(const PRope& r, int row) {
  const int i = row % r.H, half = r.hd >> 1, quads = r.nh * (half >> 2);
  const rsrc_t q = rsrc(r.qkv + (size_t)row * r.ld), qo = rsrc(r.out + (size_t)row * r.ld);
  const rsrc_t t = rsrc(r.cs + (size_t)i * r.hd);
  for (int idx = local_tid(); idx < quads; idx += 256) {
    const int h = idx / (half >> 2), d = (idx - h * (half >> 2)) * 4;
    const int o0 = (h * r.hd + d) * 2, o1 = o0 + half * 2;
    u32x2_t a, b;
    if (r.coh) {
      a = __builtin_amdgcn_raw_buffer_load_b64(q, o0, 0, COH);
      b = __builtin_amdgcn_raw_buffer_load_b64(q, o1, 0, COH);
    } else {
      a = __builtin_amdgcn_raw_buffer_load_b64(q, o0, 0, PLAIN);
      b = __builtin_amdgcn_raw_buffer_load_b64(q, o1, 0, PLAIN);
    }
    const f32x4_t c01 = ld_f4<PLAIN>(t, d * 8), c23 = ld_f4<PLAIN>(t, d * 8 + 16);
    const float cs[8] = {c01[0], c01[1], c01[2], c01[3], c23[0], c23[1], c23[2], c23[3]};
    float x[4], y[4];
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      x[2 * j] = __uint_as_float(a[j] << 16);
      x[2 * j + 1] = __uint_as_float(a[j] & 0xFFFF0000u);
      y[2 * j] = __uint_as_float(b[j] << 16);
      y[2 * j + 1] = __uint_as_float(b[j] & 0xFFFF0000u);
    }
    float u[4], v[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      u[j] = x[j] * cs[2 * j] - y[j] * cs[2 * j + 1];
      v[j] = y[j] * cs[2 * j] + x[j] * cs[2 * j + 1];
    }
    st_bf16x4(qo, (size_t)o0, u[0], u[1], u[2], u[3]);
    st_bf16x4(qo, (size_t)o1, v[0], v[1], v[2], v[3]);
  }
}

// L2 warm-up by the blocks without an item: while the other blocks work on phase p, a
// block that has no item in it touches one dword of every 128-byte line that the
// items of phase p + 1 on its XCD (item j runs on block j, XCD j % 8) read from memory
// written before the launch -- the item's weight rows, or the keys and values of a
// prefix attention split, and the shift rows of a norm, which all of them read -- so
// that those items' loads at the barrier find the lines in the XCD's L2.  The idle
// blocks of an XCD share its items round-robin; a block with an item of its own never
// issues these loads, so none of its waits include them.
template <int HD>
RAVEL_DEV void idle_warm(const Phase& nx, int items_now, const int* slots) {
  const int b = blockIdx.x, G = gridDim.x;
  if (b < items_now) return;
  const int x = b & 7;
  const int first = items_now + ((x - (items_now & 7)) + 8) % 8;  // this XCD's first idle block
  if (first >= G) return;
  const int rank = (b - first) >> 3, count = (G - 1 - first) / 8 + 1;
  const int ntype = uni(nx.type);
  const int nitems = min(uni(nx.items), G);
  const int tid = local_tid();
  unsigned acc = 0;
  if (ntype == PH_GEMM && nitems > x) {
    // the norm's shift rows, which every item of the phase reads (K/64 lines per row)
    const PGemm g = make_uniform(nx.g);
    if (g.a_mode == PA_NORM && g.shift) {
      // line l: rows 2j, 2j + 1 of 32-column tile c (tiles), or 64 columns of a row
      const int lpr = g.sh_t32 ? (g.M + 1) >> 1 : g.K >> 6, lines = (g.sh_t32 ? g.K >> 5 : g.M) * lpr;
      const rsrc_t rs = rsrc(g.shift);
      for (int l = rank * 256 + tid; l < lines; l += count * 256) {
        const size_t o = g.sh_t32 ? ((size_t)(l / lpr) * 2048 + (size_t)(l % lpr) * 64) * 2
                                  : ((size_t)(l / lpr) * g.ld_shift + (l % lpr) * 64) * 2;
        acc += __builtin_amdgcn_raw_buffer_load_b32(rs, o, 0, PLAIN);
      }
    }
  }
  for (int j = x; j < nitems; j += 8) {
    if (((j >> 3) % count) != rank) continue;
    if (ntype == PH_GEMM) {
      const PGemm g = make_uniform(nx.g);
      const int tiles = (g.N + 63) >> 6, tile = j % tiles, z = j / tiles;
      // rows and 64-column lines per row of the item's weights
      const int rows = g.wk ? 16 * g.wk : 64, lpr = g.wk ? g.K >> 6 : 4 * g.kw;
      const int n0 = g.wk ? j * rows : tile * 64, kb = g.wk ? 0 : z * 256 * g.kw;
      const rsrc_t rw = rsrc(g.W);
      for (int l = tid; l < rows * lpr; l += 256) {
        const int n = n0 + l / lpr, k = kb + (l % lpr) * 64;
        acc += __builtin_amdgcn_raw_buffer_load_b32(rw, boff(n < g.N && k < g.K, ((size_t)n * g.ldw + k) * 2), 0,
                                                    PLAIN);
      }
    } else if (ntype == PH_ATTN) {
      const AttnArgs a = make_uniform(nx.at);
      const SplitKeys k = split_keys(a, j);
      if (k.self) continue;
      constexpr int LPK = HD / 64 > 0 ? HD / 64 : 1;  // lines per key row of one head
      const int slot = a.slot ? slots[k.e] : 0;
      const int half = uni(tid >> 7);  // waves 0-1: keys, waves 2-3: values
      const bf16_t* base = (const bf16_t*)(half ? a.pv : a.pk) + slot * a.p_slot_stride + k.e * a.p_env_stride;
      const int l = tid & 127, key = k.kbeg + l / LPK, dc = (l % LPK) * 64;
      acc += __builtin_amdgcn_raw_buffer_load_b32(
          rsrc(base), boff(key < k.kend && dc < HD, ((size_t)key * a.p_ld + k.g * HD + dc) * 2), 0, PLAIN);
    }
  }
  asm volatile("" ::"v"(acc));
}

template <int MT, int HD>
__global__ __launch_bounds__(256) void persistent_step_kernel(const Phase* __restrict__ phases, int nphase,
                                                              const int* __restrict__ env_slot, int nenv,
                                                              unsigned* bar, int* err, unsigned long long* times,
                                                              unsigned* counters, int ncounters) {
  __shared__ PSmem sm;
  __shared__ Phase desc[3];
  __shared__ int slots[64];
  __shared__ int ok;
  const int tid = threadIdx.x;
  // a barrier of an earlier launch timed out and its counters are stale: do
  // nothing until the host has re-armed them (the error word is sticky until then)
  if (tid == 0) ok = __hip_atomic_load(gptr(err), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == 0;
  __syncthreads();
  if (!ok) return;
  const bool stamp = times != nullptr && blockIdx.x == 0 && tid == 0;
  if (stamp) *gptr(times) = wall_clock64();
  for (int d = 0; d < 2 && d < nphase; ++d)
    if (tid < kDescChunks)
      reinterpret_cast<u32x4_t*>(&desc[d])[tid] = *gptr(reinterpret_cast<const u32x4_t*>(&phases[d]) + tid);
  if (env_slot && tid < nenv && tid < 64) slots[tid] = *gptr(env_slot + tid);
  __syncthreads();

  // Phase p: this block's first item's reads of memory written before the launch --
  // GEMM weight fragments (16), or the keys and values (8) of a prefix attention
  // split -- are issued first, then the block waits at barrier p (between phases
  // p - 1 and p), so the fetch overlaps the wait.  (Issued any earlier, these loads
  // would sit in front of the previous phase's own loads and stores in the wave's
  // in-order memory counter, and every wait of that phase would wait for them too.)
  // The registers they land in belong to the phase's own branch of the loop.
  u32x4_t dreg = {0, 0, 0, 0};  // descriptor p + 1, loaded after arriving at barrier p
  auto wait_in = [&](int p) -> bool {
    if (p == 0) return true;
    if (tid == 0) ok = barrier_wait(bar, (unsigned)p, err);
    __syncthreads();
    if (!ok) return false;
    if (p + 1 < nphase && tid < kDescChunks) reinterpret_cast<u32x4_t*>(&desc[(p + 1) % 3])[tid] = dreg;
    if (stamp) *gptr(times + p) = wall_clock64();
    __syncthreads();
    return true;
  };

  auto none = [] {};

  for (int p = 0; p < nphase; ++p) {
    const Phase& ph = desc[p % 3];
    const int type = uni(ph.type), items = uni(ph.items);
    if (type == PH_GEMM) {
      const PGemm g = make_uniform(ph.g);
      u32x4_t pre[16];
      // whole-K norm phases: the shift fragments are staged in LDS with the prefetch
      const bool stage = g.wk > 0 && g.a_mode == PA_NORM && g.shift != nullptr;
      if ((int)blockIdx.x < items) {
        load_weights(g, blockIdx.x, pre);
        if (stage) stage_shift<MT>(g, sm);
      }
      if (!wait_in(p)) return;
      for (int item = blockIdx.x; item < items; item += gridDim.x) {
        if (item != (int)blockIdx.x) load_weights(g, item, pre);
        const bool staged = stage && item == (int)blockIdx.x;
        if (g.wk == 2)
          gemm_item_wk<MT, 2>(g, item, pre, sm, staged);
        else if (g.wk == 1)
          gemm_item_wk<MT, 1>(g, item, pre, sm, staged);
        else if (g.kw == 2)
          gemm_item<MT, 2>(g, item, pre, err, sm, none);
        else
          gemm_item<MT, 1>(g, item, pre, err, sm, none);
      }
    } else if (type == PH_ATTN) {
      const AttnArgs a = make_uniform(ph.at);
      u32x4_t kv[8];
      bool kv_ready = false;
      if ((int)blockIdx.x < items) {
        const SplitKeys k = split_keys(a, blockIdx.x);
        if (!k.self) {
          attn_load_kv_aux<HD, PLAIN>(a, k, slots, kv);
          kv_ready = true;
        }
      }
      if (!wait_in(p)) return;
      for (int item = blockIdx.x; item < items; item += gridDim.x)
        attn_item<HD>(a, item, slots, err, sm, kv, item == (int)blockIdx.x && kv_ready, none);
    } else {
      if (!wait_in(p)) return;
      if (type == PH_ROPE) {
        const PRope r = make_uniform(ph.r);
        for (int item = blockIdx.x; item < items; item += gridDim.x) rope_item(r, item);
      }
    }
    // side work of the phase for the blocks without an item, then the L2 warm-up of
    // the next phase by the blocks past those
    const int nside = uni(ph.side.nitems);
    if (nside > 0 && (int)blockIdx.x >= items && (int)blockIdx.x < items + nside) {
      const PSide sd = make_uniform(ph.side);
      side_item<MT>(sd, sd.item0 + (int)blockIdx.x - items, sm);
    }
    if (p + 1 == nphase) break;
    idle_warm<HD>(desc[(p + 1) % 3], items + nside, slots);
    // arrive at barrier p + 1 once every wave's stores are done; fetch descriptor
    // p + 2 (written to LDS after that barrier)
    wait_memory();
    __syncthreads();
    if (tid == 0) barrier_arrive(bar, (unsigned)(p + 1));
    if (p + 2 < nphase && tid < kDescChunks) dreg = *gptr(reinterpret_cast<const u32x4_t*>(&phases[p + 2]) + tid);
  }
  if (stamp) *gptr(times + nphase) = wall_clock64();
  // re-arm the barrier: the last block to get here has seen every block pass
  // every barrier, and zeroes the counters for the next launch
  wait_memory();
  __syncthreads();
  if (tid == 0) {
    unsigned* ex = bar + 64 * (2 + kBarrierGroups);
    const unsigned prev = __hip_atomic_fetch_add(gptr(ex), 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    ok = prev == gridDim.x - 1;
    if (ok) {
      for (int i = 0; i < 2 + kBarrierGroups; ++i)
        __hip_atomic_store(gptr(bar + 64 * i), 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(gptr(ex), 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
  __syncthreads();
  // ... and the split counters of every phase
  if (ok)
    for (int i = tid; i < ncounters; i += 256)
      __hip_atomic_store(gptr(counters + (size_t)i * kCounterStride), 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

template <int MT>
const void* kernel_for_hd(int hd) {
  switch (hd) {
    case 32: return (const void*)persistent_step_kernel<MT, 32>;
    case 64: return (const void*)persistent_step_kernel<MT, 64>;
    case 128: return (const void*)persistent_step_kernel<MT, 128>;
    case 256: return (const void*)persistent_step_kernel<MT, 256>;
    default: return nullptr;
  }
}

const void* kernel_for(int mt, int hd) {
  switch (mt) {
    case 1: return kernel_for_hd<1>(hd);
    case 2: return kernel_for_hd<2>(hd);
    case 4: return kernel_for_hd<4>(hd);
    default: return nullptr;
  }
}

}  // namespace

hipError_t launch_persistent(const Phase* phases, int nphase, const int* env_slot, int nenv, int mt, int hd, int blocks,
                             unsigned* bar, int* err, unsigned long long* times, unsigned* counters, int ncounters,
                             hipStream_t s) {
  const void* fn = kernel_for(mt, hd);
  if (!fn || nenv > 64 || nphase < 1 || ncounters < 0) return hipErrorInvalidValue;
  void* args[] = {(void*)&phases, (void*)&nphase, (void*)&env_slot, (void*)&nenv,     (void*)&bar,
                  (void*)&err,    (void*)&times,  (void*)&counters, (void*)&ncounters};
  // An ordinary launch: the grid (one block per CU, at most the occupancy limit)
  // is co-resident as soon as the CUs are free, and every wait in the kernel is
  // bounded, so a block held back by other work only delays the first barrier; a
  // wait that never completes sets the error word and every block leaves.
  return hipLaunchKernel(fn, dim3(blocks), dim3(256), args, 0, s);
}

int persistent_max_blocks(int mt, int hd) {
  const void* fn = kernel_for(mt, hd);
  if (!fn) return 0;
  int per_cu = 0, dev = 0, cus = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, 256, 0) != hipSuccess) return 0;
  if (hipGetDevice(&dev) != hipSuccess) return 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
  return per_cu * cus;
}

}  // namespace ravel
