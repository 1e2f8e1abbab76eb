// Attention of the buffer tokens over [prefix tokens ; buffer tokens] (and of
// the FOP adapters over FOP tokens), bidirectional, grouped-query heads.
//
// bf16 path (MFMA, wave64): one block per (key split, query head, env); each
// of the 4 waves owns 16-query blocks.  Key/value tiles of 32 keys are staged
// in LDS (V stored transposed) and shared by the waves.  Scores are computed
// transposed, S^T = K Q^T, so that each lane owns one query: the online
// softmax statistics stay in registers and P^T feeds the second MFMA
// O^T += V^T P^T directly, without an LDS round trip.  With several key
// splits, each block writes (m, l, unnormalised O) and the last block of the
// (env, head) merges the splits in fixed order.
//
// fp32 path: one wavefront per (query, head, env), lanes over head dims.
#include "kernels.h"

namespace ravel {

static constexpr float kLog2e = 1.4426950408889634f;

template <typename T>
RAVEL_DEV const T* key_base(const AttnArgs& a, const T* pbase, const T* sbase, int e, int kidx, int g,
                            int hd) {
  if (kidx < a.P) return pbase + (long long)kidx * a.p_ld + g * hd;
  return sbase + (long long)(e * a.S + (kidx - a.P)) * a.s_ld + g * hd;
}

template <int HD, int MAXQB>
__global__ __launch_bounds__(256) void attn_bf16_kernel(AttnArgs a) {
  constexpr int TK = 32;
  constexpr int KS = HD / 32;  // k-steps of the score MFMA
  constexpr int DT = HD / 16;  // 16-row tiles of O^T
  __shared__ __attribute__((aligned(16))) bf16_t Ks[TK][HD + 8];
  __shared__ __attribute__((aligned(16))) bf16_t Vt[HD][TK + 8];
  __shared__ int s_last;

  const int split = blockIdx.x, j = blockIdx.y, e = blockIdx.z;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l16 = lane & 15, grp = lane >> 4;
  const int g = (j * a.nkv) / a.nq;
  const int QB = (a.Hq + 15) / 16;
  const int nkeys = a.P + a.S;
  const int kbeg = split * a.keys_per_split;
  const int kend = min(nkeys, kbeg + a.keys_per_split);

  const bf16_t* q = (const bf16_t*)a.q;
  const int slot = a.slot ? a.slot[e] : 0;
  const bf16_t* pk = (const bf16_t*)a.pk + slot * a.p_slot_stride + e * a.p_env_stride;
  const bf16_t* pv = (const bf16_t*)a.pv + slot * a.p_slot_stride + e * a.p_env_stride;
  const bf16_t* sk = (const bf16_t*)a.sk;
  const bf16_t* sv = (const bf16_t*)a.sv;

  bf16x8_t qf[MAXQB][KS];
  f32x4_t o[MAXQB][DT];
  float mrow[MAXQB], lrow[MAXQB];
#pragma unroll
  for (int qi = 0; qi < MAXQB; ++qi) {
    const int qb = wave + 4 * qi;
    const int query = qb * 16 + l16;
    mrow[qi] = -INFINITY;
    lrow[qi] = 0.f;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) o[qi][dt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      if (qb < QB && query < a.Hq)
        qf[qi][ks] = *(const bf16x8_t*)(q + (size_t)(e * a.Hq + query) * a.ldq + j * HD + ks * 32 + grp * 8);
      else
        qf[qi][ks] = bf16x8_t{};
    }
  }
  const float sl2 = a.scale * kLog2e;

  // K/V tiles: loaded into registers one tile ahead, then written to LDS (V
  // transposed) so that global latency overlaps the previous tile's MFMAs.
  constexpr int KCH = (TK * (HD / 8) + 255) / 256;        // K chunks per thread
  constexpr int VIT = ((TK / 4) * (HD / 8) + 255) / 256;  // V items (4 keys x 8 dims) per thread
  u32x4_t kreg[KCH];
  u32x4_t vreg[VIT][4];
  auto load_tile = [&](int k0) {
#pragma unroll
    for (int i = 0; i < KCH; ++i) {
      const int c = tid + i * 256;
      const int row = c / (HD / 8), dc = (c % (HD / 8)) * 8;
      const int kidx = k0 + row;
      kreg[i] = u32x4_t{0, 0, 0, 0};
      if (c < TK * (HD / 8) && kidx < kend) kreg[i] = *(const u32x4_t*)(key_base(a, pk, sk, e, kidx, g, HD) + dc);
    }
#pragma unroll
    for (int it = 0; it < VIT; ++it) {
      const int c = tid + it * 256;
      const int kq = c / (HD / 8), dc = (c % (HD / 8)) * 8;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int kidx = k0 + kq * 4 + i;
        vreg[it][i] = u32x4_t{0, 0, 0, 0};
        if (c < (TK / 4) * (HD / 8) && kidx < kend)
          vreg[it][i] = *(const u32x4_t*)(key_base(a, pv, sv, e, kidx, g, HD) + dc);
      }
    }
  };
  auto store_tile = [&]() {
#pragma unroll
    for (int i = 0; i < KCH; ++i) {
      const int c = tid + i * 256;
      if (c < TK * (HD / 8)) *(u32x4_t*)&Ks[c / (HD / 8)][(c % (HD / 8)) * 8] = kreg[i];
    }
#pragma unroll
    for (int it = 0; it < VIT; ++it) {
      const int c = tid + it * 256;
      if (c >= (TK / 4) * (HD / 8)) continue;
      const int kq = c / (HD / 8), dc = (c % (HD / 8)) * 8;
      const bf16_t* h0 = (const bf16_t*)&vreg[it][0];
      const bf16_t* h1 = (const bf16_t*)&vreg[it][1];
      const bf16_t* h2 = (const bf16_t*)&vreg[it][2];
      const bf16_t* h3 = (const bf16_t*)&vreg[it][3];
#pragma unroll
      for (int dd = 0; dd < 8; ++dd) {
        u32x2_t w;
        w[0] = (uint32_t)h0[dd] | ((uint32_t)h1[dd] << 16);
        w[1] = (uint32_t)h2[dd] | ((uint32_t)h3[dd] << 16);
        *(u32x2_t*)&Vt[dc + dd][kq * 4] = w;
      }
    }
  };

  if (kbeg < kend) load_tile(kbeg);
  for (int k0 = kbeg; k0 < kend; k0 += TK) {
    __syncthreads();
    store_tile();
    __syncthreads();
    if (k0 + TK < kend) load_tile(k0 + TK);

#pragma unroll
    for (int qi = 0; qi < MAXQB; ++qi) {
      const int qb = wave + 4 * qi;
      if (qb >= QB) continue;  // wave-uniform
      // S^T[key][query] for two 16-key sub-tiles
      f32x4_t s[2];
#pragma unroll
      for (int st = 0; st < 2; ++st) {
        s[st] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          const bf16x8_t kf = *(const bf16x8_t*)&Ks[st * 16 + l16][ks * 32 + grp * 8];
          s[st] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf, qf[qi][ks], s[st], 0, 0, 0);
        }
      }
      float mx = -INFINITY;
#pragma unroll
      for (int st = 0; st < 2; ++st)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int kidx = k0 + st * 16 + grp * 4 + r;
          float x = s[st][r] * sl2;
          if (kidx >= kend) x = -INFINITY;
          s[st][r] = x;
          mx = fmaxf(mx, x);
        }
      mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
      mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
      const float mnew = fmaxf(mrow[qi], mx);
      const float corr = (mnew == -INFINITY) ? 1.f : exp2f(mrow[qi] - mnew);
      float psum = 0.f;
      float p[2][4];
#pragma unroll
      for (int st = 0; st < 2; ++st)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          p[st][r] = (s[st][r] == -INFINITY) ? 0.f : exp2f(s[st][r] - mnew);
          psum += p[st][r];
        }
      psum += __shfl_xor(psum, 16, 64);
      psum += __shfl_xor(psum, 32, 64);
      lrow[qi] = lrow[qi] * corr + psum;
      mrow[qi] = mnew;
      // P^T as the B operand: slot jj of group grp is key (jj<4 ? 4grp+jj : 16+4grp+jj-4)
      bf16x8_t pf;
      {
        bf16_t pb[8];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          pb[r] = f32_to_bf16(p[0][r]);
          pb[4 + r] = f32_to_bf16(p[1][r]);
        }
        pf = *(const bf16x8_t*)pb;
      }
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        o[qi][dt][0] *= corr;
        o[qi][dt][1] *= corr;
        o[qi][dt][2] *= corr;
        o[qi][dt][3] *= corr;
        const bf16_t* vrow = &Vt[dt * 16 + l16][0];
        u32x4_t vv;
        const u32x2_t lo = *(const u32x2_t*)(vrow + grp * 4);
        const u32x2_t hi = *(const u32x2_t*)(vrow + 16 + grp * 4);
        vv[0] = lo[0];
        vv[1] = lo[1];
        vv[2] = hi[0];
        vv[3] = hi[1];
        o[qi][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(*(const bf16x8_t*)&vv, pf, o[qi][dt], 0, 0, 0);
      }
    }
  }

  // o[qi][dt][r] = O^T[d = dt*16 + 4grp + r][query = qb*16 + l16]
  bf16_t* out = (bf16_t*)a.out;
  if (a.nsplit == 1) {
#pragma unroll
    for (int qi = 0; qi < MAXQB; ++qi) {
      const int qb = wave + 4 * qi;
      const int query = qb * 16 + l16;
      if (qb >= QB || query >= a.Hq) continue;
      const float inv = 1.f / lrow[qi];
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        u32x2_t w;
        w[0] = (uint32_t)f32_to_bf16(o[qi][dt][0] * inv) | ((uint32_t)f32_to_bf16(o[qi][dt][1] * inv) << 16);
        w[1] = (uint32_t)f32_to_bf16(o[qi][dt][2] * inv) | ((uint32_t)f32_to_bf16(o[qi][dt][3] * inv) << 16);
        *(u32x2_t*)(out + (size_t)(e * a.Hq + query) * a.ldo + j * HD + dt * 16 + grp * 4) = w;
      }
    }
    return;
  }

  const int Hp = QB * 16;
  const size_t pidx = ((size_t)e * a.nq + j) * a.nsplit + split;
#pragma unroll
  for (int qi = 0; qi < MAXQB; ++qi) {
    const int qb = wave + 4 * qi;
    const int query = qb * 16 + l16;
    if (qb >= QB) continue;
    float* po = a.part_o + (pidx * Hp + query) * HD;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) coherent_store4(po + dt * 16 + grp * 4, o[qi][dt]);
    if (grp == 0) {
      coherent_store(&a.part_ml[(pidx * Hp + query) * 2 + 0], mrow[qi]);
      coherent_store(&a.part_ml[(pidx * Hp + query) * 2 + 1], lrow[qi]);
    }
  }
  if (!last_block_arrival(&a.counters[(e * a.nq + j) * kCounterStride], (unsigned)a.nsplit, &s_last)) return;
  // merge the key splits in fixed order: softmax weights of every (split, query)
  // first (into LDS, reusing the K tile), then each thread owns 4 dims of a query
  const size_t pbase = ((size_t)e * a.nq + j) * a.nsplit;
  float* wgt = reinterpret_cast<float*>(&Ks[0][0]);  // [nsplit][Hq] (fits: nsplit*Hq <= TK*(HD+8)/2)
  for (int query = tid; query < a.Hq; query += 256) {
    float mmax = -INFINITY;
    for (int sp = 0; sp < a.nsplit; ++sp) mmax = fmaxf(mmax, a.part_ml[((pbase + sp) * Hp + query) * 2]);
    float den = 0.f;
    for (int sp = 0; sp < a.nsplit; ++sp) {
      const float ms = a.part_ml[((pbase + sp) * Hp + query) * 2];
      const float wv = (ms == -INFINITY) ? 0.f : exp2f(ms - mmax);
      wgt[sp * a.Hq + query] = wv;
      den += wv * a.part_ml[((pbase + sp) * Hp + query) * 2 + 1];
    }
    const float inv = 1.f / den;
    for (int sp = 0; sp < a.nsplit; ++sp) wgt[sp * a.Hq + query] *= inv;
  }
  __syncthreads();
  for (int idx = tid; idx < a.Hq * (HD / 4); idx += 256) {
    const int query = idx / (HD / 4), d = (idx % (HD / 4)) * 4;
    f32x4_t num = {0.f, 0.f, 0.f, 0.f};
#pragma unroll 4
    for (int sp = 0; sp < a.nsplit; ++sp) {
      const float wv = wgt[sp * a.Hq + query];
      const f32x4_t os = *(const f32x4_t*)&a.part_o[((pbase + sp) * Hp + query) * HD + d];
      num[0] += wv * os[0];
      num[1] += wv * os[1];
      num[2] += wv * os[2];
      num[3] += wv * os[3];
    }
    u32x2_t wv;
    wv[0] = (uint32_t)f32_to_bf16(num[0]) | ((uint32_t)f32_to_bf16(num[1]) << 16);
    wv[1] = (uint32_t)f32_to_bf16(num[2]) | ((uint32_t)f32_to_bf16(num[3]) << 16);
    *(u32x2_t*)(out + (size_t)(e * a.Hq + query) * a.ldo + j * HD + d) = wv;
  }
}

// ---------------------------------------------------------------------------
// Grouped-query form for whole-range (unsplit) attention.  The G = nq/nkv query
// heads that share one K/V head are flattened with the queries into one row
// space of G*Hq rows (row = h*Hq + query), cut into 16-row MFMA blocks; a
// block of NW waves owns NW consecutive row blocks (one per wave) of one
// (env, KV head) and streams all keys once, so each K/V tile is staged in LDS
// once for every query head of the group.  With 8 waves two share each SIMD:
// one wave's MFMAs run while the other does its softmax or waits on LDS.  K/V
// tiles are double-buffered in LDS (one barrier per tile); their global loads
// are issued two tiles ahead into registers, so about two tiles of MFMA time
// cover each load's latency.  V is written
// transposed with 8 keys x 4-lane groups per row.
//
// Softmax rescaling is lazy: the running maximum m of a row only moves when a
// tile raises it by more than kLazy (log2 units), so between moves exp2(s - m)
// <= 2^kLazy and the O rescale (a VALU pass over all accumulators) is skipped
// for the wave unless one of its rows moved.  The result is the same softmax;
// only the reference point of the bf16-rounded probabilities differs.
// ---------------------------------------------------------------------------
static constexpr float kLazy = 8.f;

template <int HD, int NW, int TK>
__global__ __launch_bounds__(NW * 64) void attn_gqa_kernel(AttnArgs a, int chunks) {
  constexpr int NT = NW * 64;
  constexpr int KS = HD / 32;
  constexpr int DT = HD / 16;
  constexpr int KLD = HD + 8;
  // V^T row stride TK / 2 + 2 dwords (18 for 32-key tiles; 20 measured slower)
  constexpr int VLD = TK + 4;
  __shared__ __attribute__((aligned(16))) bf16_t Ks[2][TK][KLD];
  __shared__ __attribute__((aligned(16))) bf16_t Vt[2][HD][VLD];

  // blocks that share an (env, KV head) sit on one XCD (dispatch is round-robin
  // over the 8 XCDs), so the group's K/V is fetched into one L2 only
  const int total = gridDim.x;
  const int L = blockIdx.x;
  const int w = (total % 8 == 0) ? (L % 8) * (total / 8) + L / 8 : L;
  const int chunk = w % chunks;
  const int g = (w / chunks) % a.nkv;
  const int e = w / (chunks * a.nkv);

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l16 = lane & 15, grp = lane >> 4;
  const int G = a.nq / a.nkv;
  const int R = G * a.Hq;
  const int row = (chunk * NW + wave) * 16 + l16;  // this lane's row
  // a wave whose 16 rows all lie past the group stages tiles and meets the
  // barriers but does no MFMA or softmax work (uniform per wave)
  const bool active = (chunk * NW + wave) * 16 < R;

  const bf16_t* q = (const bf16_t*)a.q;
  const int slot = a.slot ? a.slot[e] : 0;
  const bf16_t* pk = (const bf16_t*)a.pk + slot * a.p_slot_stride + e * a.p_env_stride;
  const bf16_t* pv = (const bf16_t*)a.pv + slot * a.p_slot_stride + e * a.p_env_stride;
  const bf16_t* sk = (const bf16_t*)a.sk;
  const bf16_t* sv = (const bf16_t*)a.sv;

  // rows past the group are clamped to a real row, computed and never stored
  bf16x8_t qf[KS];
  {
    const int r = min(row, R - 1);
    const int h = r / a.Hq, query = r % a.Hq;
    const bf16_t* qr = q + (size_t)(e * a.Hq + query) * a.ldq + (g * G + h) * HD + grp * 8;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) qf[ks] = *(const bf16x8_t*)(qr + ks * 32);
  }
  f32x4_t o[DT];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt) o[dt] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  float mrow = -INFINITY, lrow = 0.f;
  const float sl2 = a.scale * kLog2e;

  // K: 16-byte chunks, row-major.  V: items of 4 keys x 8 dims, kq fastest so
  // that 8 lanes fill one 64-byte row segment of V^T.  Keys past the range are
  // clamped to the last key: finite values whose probabilities are exactly 0.
  constexpr int KCHUNKS = TK * (HD / 8), VITEMS = (TK / 4) * (HD / 8);
  constexpr int KCH = (KCHUNKS + NT - 1) / NT;
  constexpr int VIT = (VITEMS + NT - 1) / NT;
  // Two register sets: tile j is fetched into set j % 2 two tiles ahead of its
  // MFMAs and written to LDS one tile ahead, so each load has about two tiles
  // of MFMA time to arrive.
  struct Stage {
    u32x4_t k[KCH];
    u32x4_t v[VIT][4];
  };
  Stage st0, st1;
  // Key tiles: the prefix rows padded to a multiple of TK, then the buffer's own
  // rows, so that every tile reads one part from one uniform base.  Rows past a
  // part's end are clamped to its last row (finite values) and masked out of
  // the softmax.
  const int Ppad = ((a.P + TK - 1) / TK) * TK;
  const bf16_t* sk_e = sk + (size_t)e * a.S * a.s_ld;
  const bf16_t* sv_e = sv + (size_t)e * a.S * a.s_ld;
  auto load_tile = [&](int k0, Stage& sg) {
    const bool pre = k0 < Ppad;  // uniform
    const int r0 = pre ? k0 : k0 - Ppad;
    const int last = (pre ? a.P : a.S) - 1;
    const int ld = pre ? a.p_ld : a.s_ld;
    const bf16_t* kb = (pre ? pk : sk_e) + g * HD;
    const bf16_t* vb = (pre ? pv : sv_e) + g * HD;
#pragma unroll
    for (int i = 0; i < KCH; ++i) {
      const int c = tid + i * NT;
      if (KCHUNKS % NT == 0 || c < KCHUNKS) {
        const int r = min(r0 + c / (HD / 8), last);
        sg.k[i] = *(const u32x4_t*)(kb + (size_t)r * ld + (c % (HD / 8)) * 8);
      }
    }
#pragma unroll
    for (int it = 0; it < VIT; ++it) {
      const int c = tid + it * NT;
      if (VITEMS % NT == 0 || c < VITEMS) {
        const int kq = c % (TK / 4), dc = (c / (TK / 4)) * 8;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int r = min(r0 + kq * 4 + i, last);
          sg.v[it][i] = *(const u32x4_t*)(vb + (size_t)r * ld + dc);
        }
      }
    }
  };
  auto store_tile = [&](int buf, const Stage& sg) {
#pragma unroll
    for (int i = 0; i < KCH; ++i) {
      const int c = tid + i * NT;
      if (KCHUNKS % NT == 0 || c < KCHUNKS) *(u32x4_t*)&Ks[buf][c / (HD / 8)][(c % (HD / 8)) * 8] = sg.k[i];
    }
#pragma unroll
    for (int it = 0; it < VIT; ++it) {
      const int c = tid + it * NT;
      if (VITEMS % NT == 0 || c < VITEMS) {
        const int kq = c % (TK / 4), dc = (c / (TK / 4)) * 8;
#pragma unroll
        for (int m = 0; m < 4; ++m) {
          const uint32_t a0 = sg.v[it][0][m], a1 = sg.v[it][1][m];
          const uint32_t a2 = sg.v[it][2][m], a3 = sg.v[it][3][m];
          // dims dc+2m (low halves of a0..a3) and dc+2m+1 (high halves), one byte
          // permute per output word
          u32x2_t lo, hi;
          lo[0] = __builtin_amdgcn_perm(a1, a0, 0x05040100u);
          lo[1] = __builtin_amdgcn_perm(a3, a2, 0x05040100u);
          hi[0] = __builtin_amdgcn_perm(a1, a0, 0x07060302u);
          hi[1] = __builtin_amdgcn_perm(a3, a2, 0x07060302u);
          *(u32x2_t*)&Vt[buf][dc + 2 * m][kq * 4] = lo;
          *(u32x2_t*)&Vt[buf][dc + 2 * m + 1][kq * 4] = hi;
        }
      }
    }
  };

  const int ntile = Ppad / TK + (a.S + TK - 1) / TK;
  load_tile(0, st0);
  if (1 < ntile) load_tile(TK, st1);
  store_tile(0, st0);
  __syncthreads();
  // tile t: fetch tile t + 2 into the set tile t came from, MFMAs on LDS buffer
  // t & 1, write tile t + 1 (the other set) into the other buffer
  auto tile_step = [&](int t, Stage& s_next2, const Stage& s_next1) {
    const int k0 = t * TK, buf = t & 1;
    if (t + 2 < ntile) load_tile(k0 + 2 * TK, s_next2);
    if (active) {
    // S^T[key][row] for the tile's NS 16-key sub-tiles, each summed in two
    // independent MFMA chains (even / odd k-steps)
    constexpr int NS = TK / 16;
    f32x4_t sa[NS], sb[NS];
#pragma unroll
    for (int u = 0; u < NS; ++u) sa[u] = sb[u] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    // the wave issuing MFMAs goes first; the SIMD's other wave fills the gaps
    // with its softmax or staging work
    __builtin_amdgcn_s_setprio(1);
#pragma unroll
    for (int ks = 0; ks < KS; ks += 2) {
#pragma unroll
      for (int u = 0; u < NS; ++u) {
        const bf16x8_t kf = *(const bf16x8_t*)&Ks[buf][u * 16 + l16][ks * 32 + grp * 8];
        sa[u] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf, qf[ks], sa[u], 0, 0, 0);
      }
      if (ks + 1 < KS) {
#pragma unroll
        for (int u = 0; u < NS; ++u) {
          const bf16x8_t kf = *(const bf16x8_t*)&Ks[buf][u * 16 + l16][(ks + 1) * 32 + grp * 8];
          sb[u] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf, qf[ks + 1], sb[u], 0, 0, 0);
        }
      }
    }
    __builtin_amdgcn_s_setprio(0);
    float x[4 * NS];
#pragma unroll
    for (int u = 0; u < NS; ++u)
#pragma unroll
      for (int r = 0; r < 4; ++r) x[4 * u + r] = (sa[u][r] + sb[u][r]) * sl2;
    // valid keys of the tile (uniform): the last tile of each part is ragged
    const int nvalid = k0 < Ppad ? a.P - k0 : a.S - (k0 - Ppad);
    if (nvalid < TK) {
#pragma unroll
      for (int u = 0; u < NS; ++u)
#pragma unroll
        for (int r = 0; r < 4; ++r)
          if (u * 16 + grp * 4 + r >= nvalid) x[4 * u + r] = -INFINITY;
    }
    float lmx = x[0];
#pragma unroll
    for (int r = 1; r < 4 * NS; ++r) lmx = fmaxf(lmx, x[r]);
    if (__any(lmx > mrow + kLazy)) {
      float mx = fmaxf(lmx, __shfl_xor(lmx, 16, 64));
      mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
      const float mnew = mx > mrow + kLazy ? mx : mrow;
      const float corr = exp2f(mrow - mnew);
      mrow = mnew;
      lrow *= corr;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
        o[dt][0] *= corr;
        o[dt][1] *= corr;
        o[dt][2] *= corr;
        o[dt][3] *= corr;
      }
    }
    float p[4 * NS];
#pragma unroll
    for (int r = 0; r < 4 * NS; ++r) p[r] = __builtin_amdgcn_exp2f(x[r] - mrow);
#pragma unroll
    for (int h = 0; h < NS / 2; ++h)
      lrow += ((p[8 * h] + p[8 * h + 1]) + (p[8 * h + 2] + p[8 * h + 3])) +
              ((p[8 * h + 4] + p[8 * h + 5]) + (p[8 * h + 6] + p[8 * h + 7]));
    // P^T as the B operand, one per 32 keys: slot jj of group grp is key
    // 32 h + (jj < 4 ? 4 grp + jj : 16 + 4 grp + jj - 4)
    bf16x8_t pf[NS / 2];
#pragma unroll
    for (int h = 0; h < NS / 2; ++h) {
      const u32x4_t pw = {pack_bf16x2(p[8 * h], p[8 * h + 1]), pack_bf16x2(p[8 * h + 2], p[8 * h + 3]),
                          pack_bf16x2(p[8 * h + 4], p[8 * h + 5]), pack_bf16x2(p[8 * h + 6], p[8 * h + 7])};
      pf[h] = __builtin_bit_cast(bf16x8_t, pw);
    }
    __builtin_amdgcn_s_setprio(1);
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) {
      const bf16_t* vrow = &Vt[buf][dt * 16 + l16][0];
#pragma unroll
      for (int h = 0; h < NS / 2; ++h) {
        const u32x2_t lo = *(const u32x2_t*)(vrow + 32 * h + grp * 4);
        const u32x2_t hi = *(const u32x2_t*)(vrow + 32 * h + 16 + grp * 4);
        const u32x4_t vv = {lo[0], lo[1], hi[0], hi[1]};
        o[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, vv), pf[h], o[dt], 0, 0, 0);
      }
    }
    __builtin_amdgcn_s_setprio(0);
    }
    if (t + 1 < ntile) store_tile(buf ^ 1, s_next1);
    __syncthreads();
  };
  for (int t = 0; t < ntile; t += 2) {
    tile_step(t, st0, st1);
    if (t + 1 < ntile) tile_step(t + 1, st1, st0);
  }

  // o[dt][r] = O^T[d = dt*16 + 4grp + r][row]
  lrow += __shfl_xor(lrow, 16, 64);
  lrow += __shfl_xor(lrow, 32, 64);
  if (row >= R) return;
  const int h = row / a.Hq, query = row % a.Hq;
  const float inv = 1.f / lrow;
  bf16_t* orow = (bf16_t*)a.out + (size_t)(e * a.Hq + query) * a.ldo + (g * G + h) * HD + grp * 4;
#pragma unroll
  for (int dt = 0; dt < DT; ++dt) {
    u32x2_t wv;
    wv[0] = pack_bf16x2(o[dt][0] * inv, o[dt][1] * inv);
    wv[1] = pack_bf16x2(o[dt][2] * inv, o[dt][3] * inv);
    *(u32x2_t*)(orow + dt * 16) = wv;
  }
}

template <int HD, int NW>
static hipError_t launch_gqa(const AttnArgs& a, hipStream_t s) {
  const int rb = (a.nq / a.nkv * a.Hq + 15) / 16;
  const int chunks = (rb + NW - 1) / NW;
  // key tiles of 64 where two blocks' staging still fits a CU's LDS (head dims up to
  // 128; measured ~2% faster for the 128-dim expert), of 32 otherwise
  constexpr int TK = HD <= 128 ? 64 : 32;
  hipLaunchKernelGGL((attn_gqa_kernel<HD, NW, TK>), dim3(chunks * a.nkv * a.B), dim3(NW * 64), 0, s, a, chunks);
  return hipGetLastError();
}

template <int HD, int MAXQB>
static hipError_t launch_hd(const AttnArgs& a, hipStream_t s) {
  dim3 grid(a.nsplit, a.nq, a.B);
  hipLaunchKernelGGL((attn_bf16_kernel<HD, MAXQB>), grid, dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_attn_bf16(const AttnArgs& a, hipStream_t s) {
  const int QB = (a.Hq + 15) / 16;
  if (QB > 8) return hipErrorInvalidValue;
  // the split merge keeps nsplit x Hq weights in the K tile's LDS (32 x (hd + 8) bf16)
  if (a.nsplit > 1 && a.nsplit * a.Hq > 32 * (a.hd + 8) / 2) return hipErrorInvalidValue;
  if (a.nsplit == 1 && a.nkv > 0 && a.nq % a.nkv == 0 && a.P + a.S > 0) {
    // whole key range: grouped-query kernel, 8 waves once the group has at
    // least 8 row blocks
    const bool eight = (a.nq / a.nkv * a.Hq + 15) / 16 >= 8;
    switch (a.hd) {
      case 32: return eight ? launch_gqa<32, 8>(a, s) : launch_gqa<32, 4>(a, s);
      case 64: return eight ? launch_gqa<64, 8>(a, s) : launch_gqa<64, 4>(a, s);
      case 128: return eight ? launch_gqa<128, 8>(a, s) : launch_gqa<128, 4>(a, s);
      case 256: return eight ? launch_gqa<256, 8>(a, s) : launch_gqa<256, 4>(a, s);
      default: return hipErrorInvalidValue;
    }
  }
  const bool two = QB > 4;
  switch (a.hd) {
    case 32: return two ? launch_hd<32, 2>(a, s) : launch_hd<32, 1>(a, s);
    case 64: return two ? launch_hd<64, 2>(a, s) : launch_hd<64, 1>(a, s);
    case 128: return two ? launch_hd<128, 2>(a, s) : launch_hd<128, 1>(a, s);
    case 256: return two ? launch_hd<256, 2>(a, s) : launch_hd<256, 1>(a, s);
    default: return hipErrorInvalidValue;
  }
}

// ---------------------------------------------------------------------------
// fp32 path
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(64) void attn_f32_kernel(AttnArgs a) {
  const int query = blockIdx.x, j = blockIdx.y, e = blockIdx.z;
  const int lane = threadIdx.x;
  const int hd = a.hd;
  const int g = (j * a.nkv) / a.nq;
  const int slot = a.slot ? a.slot[e] : 0;
  const float* pk = (const float*)a.pk + slot * a.p_slot_stride + e * a.p_env_stride;
  const float* pv = (const float*)a.pv + slot * a.p_slot_stride + e * a.p_env_stride;
  const float* sk = (const float*)a.sk;
  const float* sv = (const float*)a.sv;
  const float* q = (const float*)a.q + (size_t)(e * a.Hq + query) * a.ldq + j * hd;
  float qv[4], ov[4];
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    const int d = lane + 64 * c;
    qv[c] = d < hd ? q[d] : 0.f;
    ov[c] = 0.f;
  }
  float m = -INFINITY, l = 0.f;
  const int nkeys = a.P + a.S;
  for (int kidx = 0; kidx < nkeys; ++kidx) {
    const float* kr = key_base(a, pk, sk, e, kidx, g, hd);
    const float* vr = key_base(a, pv, sv, e, kidx, g, hd);
    float part = 0.f;
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int d = lane + 64 * c;
      if (d < hd) part += qv[c] * kr[d];
    }
    const float sc = wave_sum(part) * a.scale;
    const float mnew = fmaxf(m, sc);
    const float corr = expf(m - mnew);
    const float p = expf(sc - mnew);
    l = l * corr + p;
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int d = lane + 64 * c;
      ov[c] = ov[c] * corr + (d < hd ? p * vr[d] : 0.f);
    }
    m = mnew;
  }
  float* out = (float*)a.out + (size_t)(e * a.Hq + query) * a.ldo + j * hd;
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    const int d = lane + 64 * c;
    if (d < hd) out[d] = ov[c] / l;
  }
}

hipError_t launch_attn_f32(const AttnArgs& a, hipStream_t s) {
  if (a.hd > 256) return hipErrorInvalidValue;
  dim3 grid(a.Hq, a.nq, a.B);
  hipLaunchKernelGGL(attn_f32_kernel, grid, dim3(64), 0, s, a);
  return hipGetLastError();
}

}  // namespace ravel
