// libravel runtime: model creation, rolling buffers, the asynchronous context
// plane, step orchestration and hipGraph replay behind the C ABI of ravel.h.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <array>
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <map>
#include <mutex>
#include <string>
#include <vector>

#include "kernels.h"
#include "persistent.h"
#include "ravel.h"

using namespace ravel;

namespace {

thread_local std::string g_err;

ravel_status fail(ravel_status s, const std::string& msg) {
  g_err = msg;
  return s;
}

#define HIP_TRY(expr)                                                                        \
  do {                                                                                       \
    hipError_t e_ = (expr);                                                                  \
    if (e_ != hipSuccess) return fail(RAVEL_E_HIP, std::string(#expr) + ": " + hipGetErrorString(e_)); \
  } while (0)

#define RV_TRY(expr)                      \
  do {                                    \
    ravel_status s_ = (expr);             \
    if (s_ != RAVEL_OK) return s_;        \
  } while (0)

size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// Simple bump allocator over one device allocation.
struct Arena {
  size_t off = 0;
  std::vector<std::pair<void**, size_t>> pending;
  void want(void** p, size_t bytes) {
    pending.push_back({p, off});
    off = align_up(off + std::max<size_t>(bytes, 1), 256);
  }
  ravel_status commit(void** base) {
    if (hipMalloc(base, std::max<size_t>(off, 256)) != hipSuccess)
      return fail(RAVEL_E_NOMEM, "hipMalloc of " + std::to_string(off) + " bytes failed");
    for (auto& pr : pending) *pr.first = (char*)*base + pr.second;
    pending.clear();
    return RAVEL_OK;
  }
};

struct KernelRecorder {
  hipStream_t stream;
  struct Rec {
    std::string name;
    double bytes, flops;
    hipEvent_t a, b;
  };
  std::vector<Rec> recs;
  void begin(const char* name, double bytes, double flops) {
    Rec r{name, bytes, flops, nullptr, nullptr};
    (void)hipEventCreate(&r.a);
    (void)hipEventCreate(&r.b);
    (void)hipEventRecord(r.a, stream);
    recs.push_back(r);
  }
  void end() { (void)hipEventRecord(recs.back().b, stream); }
};

}  // namespace

// ---------------------------------------------------------------------------
// Model
// ---------------------------------------------------------------------------
struct LayerW {
  void* mod_w = nullptr;
  float* mod_b = nullptr;
  void* qkv_w = nullptr;
  void* o_w = nullptr;
  void* gu_w = nullptr;  // [2F, w], gate/up interleaved in blocks of 16 rows
  void* down_w = nullptr;
  int adapter = -1;  // index into the adapter list, -1 = none
  float* gamma = nullptr;
  void* qa_w = nullptr;
  void* oa_w = nullptr;
  float* alpha = nullptr;
};

struct ravel_model {
  ravel_config cfg;
  bool bf16 = true;
  size_t elt = 2;
  int device = 0;
  void* arena = nullptr;
  size_t arena_bytes = 0;
  int64_t weight_bytes = 0;
  float *in_w = nullptr, *in_b = nullptr;
  float* in_wT = nullptr;  // [D_in, w]: in_w transposed (input projection reads it); D_in = D (+1: offset column)
  float* ctau = nullptr;  // [H, w]
  void *t_w1 = nullptr, *t_w2 = nullptr;  // flow-time MLP (model dtype), kept for other step counts
  float *t_b1 = nullptr, *t_b2 = nullptr;
  float *d_w1 = nullptr, *d_b1 = nullptr, *d_b2 = nullptr;
  void* d_w2 = nullptr;
  std::vector<LayerW> layers;
  int n_ad = 0;
  void* kva_w = nullptr;  // [n_ad * 2 kvd, w]
  void* fmod_w = nullptr;  // [2w, w]
  float* fmod_b = nullptr;
  void* out_w = nullptr;
  float* out_b = nullptr;
  void* mod_all_w = nullptr;   // [(6L + 2) w, w]: every layer's modulation rows, then the final norm's
  float* mod_all_b = nullptr;  // [(6L + 2) w]
  bool has_fop_encoder = false;
  void* f_w1 = nullptr;
  float* f_b1 = nullptr;
  void* f_w2 = nullptr;
  float* f_b2 = nullptr;
  float* analytic = nullptr;
  // DynamicVLA-style offset form: action-time MLP (first layer's inputs padded to at_kz
  // columns: [e ; emb(tau) ; delta ; 0 ...]) and the offset adapter (bottleneck w/4)
  void *at_w1 = nullptr, *at_w2 = nullptr, *ta_w1 = nullptr, *ta_w2 = nullptr;
  float *at_b1 = nullptr, *at_b2 = nullptr, *ta_b1 = nullptr, *ta_alpha = nullptr;
  int at_kz = 0;
  float* rope_cs = nullptr;  // [H][hd/2][2] cos, sin of slot i's rotary angles (rope_base > 0)
};

namespace {

struct TensorMap {
  std::map<std::string, const ravel_tensor*> m;
  const ravel_tensor* get(const std::string& n) const {
    auto it = m.find(n);
    return it == m.end() ? nullptr : it->second;
  }
};

ravel_status check_shape(const ravel_tensor* t, const std::string& name, std::vector<int64_t> dims) {
  if (!t) return fail(RAVEL_E_STATE, "missing weight '" + name + "'");
  if (t->rank != (int)dims.size()) return fail(RAVEL_E_SHAPE, "weight '" + name + "': wrong rank");
  for (size_t i = 0; i < dims.size(); ++i)
    if (t->dims[i] != dims[i])
      return fail(RAVEL_E_SHAPE, "weight '" + name + "': dim " + std::to_string(i) + " is " +
                                     std::to_string(t->dims[i]) + ", expected " + std::to_string(dims[i]));
  if (!t->data) return fail(RAVEL_E_INVALID, "weight '" + name + "': null data");
  if (t->dtype != RAVEL_F32 && t->dtype != RAVEL_BF16)
    return fail(RAVEL_E_INVALID, "weight '" + name + "': unknown dtype");
  return RAVEL_OK;
}

int64_t numel(const ravel_tensor* t) {
  int64_t n = 1;
  for (int i = 0; i < t->rank; ++i) n *= t->dims[i];
  return n;
}

// Device staging for uploads: an fp32 region and a bf16 region of S elements each.
struct Staging {
  float* f = nullptr;
  bf16_t* h = nullptr;
  size_t S = 0;
};

// Upload rows [row0, row0+nrows) of a [*, cols] tensor, converting to the model
// dtype, placing source row r at destination row dst_row(r) (runs of consecutive
// destination rows are copied at once).
template <typename MapFn>
ravel_status upload_rows(const ravel_tensor* t, int64_t row0, int64_t nrows, int64_t cols, bool to_bf16,
                         void* dst, MapFn dst_row, const Staging& stg) {
  const size_t src_elt = t->dtype == RAVEL_BF16 ? 2 : 4;
  const size_t dst_elt = to_bf16 ? 2 : 4;
  if (t->dtype == RAVEL_BF16 && !to_bf16)
    return fail(RAVEL_E_INVALID, std::string(t->name) + ": bf16 source for an fp32 model");
  const int64_t chunk_rows = std::max<int64_t>(1, (int64_t)(stg.S / std::max<int64_t>(cols, 1)));
  for (int64_t r = 0; r < nrows; r += chunk_rows) {
    const int64_t nr = std::min(chunk_rows, nrows - r);
    const char* src = (const char*)t->data + (size_t)(row0 + r) * cols * src_elt;
    const void* tmp = stg.f;
    if (t->dtype == RAVEL_F32 && to_bf16) {
      HIP_TRY(hipMemcpy(stg.f, src, (size_t)nr * cols * 4, hipMemcpyDefault));
      HIP_TRY(launch_convert<bf16_t>(stg.f, stg.h, nr * cols, 0));
      tmp = stg.h;
    } else {
      HIP_TRY(hipMemcpy(stg.f, src, (size_t)nr * cols * src_elt, hipMemcpyDefault));
    }
    int64_t i = 0;
    while (i < nr) {
      int64_t j = i + 1;
      while (j < nr && dst_row(r + j) == dst_row(r + i) + (j - i)) ++j;
      HIP_TRY(hipMemcpy((char*)dst + (size_t)dst_row(r + i) * cols * dst_elt,
                        (const char*)tmp + (size_t)i * cols * dst_elt, (size_t)(j - i) * cols * dst_elt,
                        hipMemcpyDeviceToDevice));
      i = j;
    }
  }
  return RAVEL_OK;
}

ravel_status upload_all(const ravel_tensor* t, bool to_bf16, void* dst, const Staging& stg) {
  const int64_t n = numel(t);
  if (t->dtype == RAVEL_BF16 && !to_bf16)
    return fail(RAVEL_E_INVALID, std::string(t->name) + ": bf16 source for an fp32 model");
  if (!(t->dtype == RAVEL_F32 && to_bf16)) {
    HIP_TRY(hipMemcpy(dst, t->data, (size_t)n * (t->dtype == RAVEL_BF16 ? 2 : 4), hipMemcpyDefault));
    return RAVEL_OK;
  }
  if ((size_t)n <= stg.S) {
    HIP_TRY(hipMemcpy(stg.f, t->data, (size_t)n * 4, hipMemcpyDefault));
    HIP_TRY(launch_convert<bf16_t>(stg.f, (bf16_t*)dst, n, 0));
    return RAVEL_OK;
  }
  const int64_t cols = t->rank >= 2 ? t->dims[t->rank - 1] : n;
  return upload_rows(t, 0, n / cols, cols, to_bf16, dst, [](int64_t r) { return r; }, stg);
}

// GEMM dispatch ---------------------------------------------------------------
struct GemmPlan {
  bool skinny;
  bool regstream;
  bool wholek;  // skinny: 32-column blocks over the whole K (no split)
  int nfr;     // skinny: 16-column fragments per wave
  int tile;    // tiled: GemmTile
  int ksplit;
  int kchunk;
  int tiles;
  size_t part_elems;  // split-K workspace (floats)
};

// RAVEL_NO_WHOLE_K_GEMM=1: few-row GEMMs with K <= 1024 split K across blocks
// (register streaming) instead of one block per 32 columns over the whole K
bool no_wholek() {
  static const bool v = [] {
    const char* e = getenv("RAVEL_NO_WHOLE_K_GEMM");
    return e && atoi(e) != 0;
  }();
  return v;
}

GemmPlan plan_gemm(int M, int N, int K, bool geglu) {
  GemmPlan p;
  memset(&p, 0, sizeof p);
  if (M <= 64) {
    // weight streaming (measured on MI355X at the pi-style batch-1 shapes):
    //  * many column tiles and K <= 1024: one block per tile, whole K, LDS-staged rows;
    //  * otherwise: register streaming, waves split a 512 (or 256) wide K range.
    p.skinny = true;
    const int tiles64 = (N + 63) / 64;
    if (!geglu && K <= 1024 && tiles64 >= 512) {
      p.regstream = false;
      p.nfr = 1;
      p.tiles = tiles64;
      p.kchunk = K <= 128 ? 128 : K <= 256 ? 256 : K <= 512 ? 512 : 1024;
      p.ksplit = 1;
      p.part_elems = 0;
      return p;
    }
    if (!geglu && K <= 1024 && K % 128 == 0 && !no_wholek()) {
      p.regstream = false;
      p.wholek = true;
      p.tiles = (N + 31) / 32;
      p.kchunk = K;
      p.ksplit = 1;
      p.part_elems = 0;
      return p;
    }
    p.regstream = true;
    p.tiles = tiles64;
    // K ranges of 512 (8 waves per block), or of 256 when that leaves fewer blocks than CUs
    p.kchunk = (K >= 512 && (size_t)tiles64 * ((K + 511) / 512) >= 256) ? 512 : 256;
    p.ksplit = (K + p.kchunk - 1) / p.kchunk;
    const size_t tile_elems = (size_t)((M + 15) / 16) * 1024;
    p.part_elems = p.ksplit > 1 ? (size_t)p.ksplit * p.tiles * tile_elems : 0;
    return p;
  }
  // tile by shape (direct-to-LDS kernels, measured on MI355X at M = 3200, the
  // pi-style batch-64 rows: 128x128 744-804 TF/s at K = 1024; 128x64 514 and 581
  // TF/s at N = 1024, K = 2048 and 4096, where 128x128 gives 200 tiles)
  int bm, bn;
  if (M <= 256) {
    p.tile = TILE_64x128; bm = 64; bn = 128;
  } else if (N <= 1024) {
    p.tile = TILE_128x64; bm = 128; bn = 64;
  } else {
    p.tile = TILE_128x128; bm = 128; bn = 128;
  }
  p.tiles = ((M + bm - 1) / bm) * ((N + bn - 1) / bn);
  // many rows: enough tiles without splitting K (measured: split-K partial traffic
  // costs more than the wave quantisation it removes); split only tiny grids
  int ks = 1;
  while (p.tiles * ks < 128 && (K / (ks * 2)) >= 512 && ks < 8) ks *= 2;
  int kchunk = (K + ks - 1) / ks;
  kchunk = (kchunk + 63) / 64 * 64;
  p.ksplit = (K + kchunk - 1) / kchunk;
  p.kchunk = kchunk;
  p.part_elems = p.ksplit > 1 ? (size_t)p.ksplit * p.tiles * bm * bn : 0;
  return p;
}

}  // namespace

// ---------------------------------------------------------------------------
// Buffer
// ---------------------------------------------------------------------------
struct PendingCtx {
  bool valid = false;
  int64_t t_obs = 0;
  hipEvent_t ready = nullptr;
};

struct GraphEntry {
  const void* fop;
  const float* state;
  float* action;
  bool persistent;
  hipGraph_t graph;
  hipGraphExec_t exec;
};

struct ravel_buffer {
  ravel_model* m = nullptr;
  int B = 0;
  uint64_t seed = 0;
  void* arena = nullptr;
  // device state
  float* X = nullptr;
  int64_t* t = nullptr;
  int64_t* t_obs = nullptr;
  int* slot = nullptr;
  unsigned* ticket = nullptr;
  void* ctx_k = nullptr;
  void* ctx_v = nullptr;
  size_t ctx_elems = 0;  // per env per slot: L * P * nkv * hd
  // activations
  float* x = nullptr;
  void* cond = nullptr;
  void* h1 = nullptr;
  float* dvec = nullptr;  // [B, w] offset embedding d = W_d2 h1 + b_d2
  double* dval = nullptr;  // [B] offsets delta_e (RAVEL_OFFSET_CONCAT, RAVEL_OFFSET_ADAPTER)
  void* tz = nullptr;      // [BH, at_kz] inputs of the offset form's action-time MLP and adapter
  void* th = nullptr;      // [BH, w] their hidden rows
  bf16_t* pshift = nullptr;  // persistent step: bf16 copies of the norm shifts, 32-column tiles
  float* mod = nullptr;
  void* y = nullptr;
  void* qkv = nullptr;
  void* att = nullptr;
  void* qa = nullptr;
  void* kva = nullptr;
  void* u = nullptr;
  float* v = nullptr;
  float* fmod = nullptr;
  void* fhid = nullptr;
  void* obs_t = nullptr;
  float* gpart = nullptr;
  unsigned* gcnt = nullptr;
  size_t gpart_elems = 0;
  int gcnt_n = 0;
  float* apart_o = nullptr;
  float* apart_ml = nullptr;
  unsigned* acnt = nullptr;
  int* dbg_flag = nullptr;
  int attn_nsplit = 1, attn_kps = 0;
  bool mod_all = false;
  int mod_ld = 0;
  // persistent step: the modulation of layers 1 .. L - 1 and of the final norm (and
  // their bf16 shift copies) is computed inside the layer kernel by otherwise idle
  // blocks; before the launch only layer 0's
  bool side_mod = false;
  bool fused_prologue = true;  // the batch-1 step's two-launch prologue where it applies
  // per-layer modulation on the rows of distinct offset conditionings only
  bool cgroups = false;
  int* cgrp = nullptr;     // [B] conditioning group of each env (negative: not the group's first env)
  int* crowmap = nullptr;  // [B*H] modulation row of each buffer row
  int* crows = nullptr;    // (#groups) * H
  // persistent few-row path
  bool persistent = false;
  std::vector<Phase> phases;
  Phase* d_phases = nullptr;
  unsigned* pbar = nullptr;
  int* perr = nullptr;
  float* sumsq[2] = {nullptr, nullptr};
  bf16_t* pnorm = nullptr;             // p = bf16((1 + scale) * x) of the first norm, [w/32][64][32]
  std::vector<void*> pallocs;          // device memory of the persistent path
  // split tickets of the persistent kernel (re-armed with the barrier after a failure)
  unsigned* pgcnt = nullptr;  // split counters of the persistent step's phases (pcnt_n of them)
  size_t pgcnt_bytes = 0;
  int pcnt_n = 0;
  // pinned host word raised by the release kernel when the layers' kernel failed
  // (read by the next step call without synchronising), and its device address
  int* hflag = nullptr;
  int* hflag_dev = nullptr;
  int pblocks = 0, pmt = 4;
  double p_bytes = 0, p_flops = 0;
  // per phase: class name and algorithmic bytes / flops; device time stamps
  std::vector<std::string> pnames;
  std::vector<double> ph_bytes, ph_flops;
  unsigned long long* ptimes = nullptr;
  // host
  int64_t t_host = 0;
  std::vector<int> active;
  std::vector<int> has_ctx;
  std::vector<int64_t> tobs_host;
  std::vector<PendingCtx> pending;
  std::vector<hipEvent_t> retire;
  std::vector<int> retire_valid;
  std::vector<std::array<int64_t, 3>> log;
  std::mutex mu;
  bool sync_ctx = false, use_graph = true, debug = false;
  hipStream_t cap_stream = nullptr;
  std::vector<GraphEntry> graphs;
  std::map<int, float*> full_tables;  // flow-time conditioning per full-horizon step count
  float* trainX = nullptr;  // [B, H, D] training buffer of ravel_train_loss
  // relative actions: mask [D] (1 = relative dimension), state the buffer was last
  // expressed against [B, D], whether an env has one [B]
  bool relative = false;
  float* rel_mask = nullptr;
  float* s_prev = nullptr;
  int* has_prev = nullptr;
};

namespace {

template <typename T>
ravel_status run_gemm(ravel_buffer* b, hipStream_t s, KernelRecorder* rec, const char* name, const void* A,
                      int lda, const void* W, int ldb, int M, int N, int K, GemmArgs epi) {
  ravel_model* m = b->m;
  epi.A = A;
  epi.lda = lda;
  epi.B = W;
  epi.ldb = ldb;
  epi.M = M;
  epi.N = N;
  epi.K = K;
  const double elt = (double)m->elt;
  double obytes = (double)M * N * (epi.mode == EPI_F32 ? 4 : elt);
  if (epi.mode == EPI_RESID) obytes = (double)M * N * 12;  // read x, gate; write x
  if (epi.mode == EPI_RESID_TANH) obytes = (double)M * N * 8;
  if (epi.mode == EPI_GEGLU) obytes = (double)M * (N / 2) * elt;
  if (epi.mode == EPI_COND) obytes = (double)M * m->cfg.horizon * N * elt;
  const double bytes = ((double)M * K + (double)N * K) * elt + obytes;
  const double flops = 2.0 * M * N * K;
  if (!m->bf16) {
    epi.ksplit = 1;
    epi.kchunk = K;
    if (rec) rec->begin(name, epi.m_rows ? 0.0 : bytes, epi.m_rows ? 0.0 : flops);
    HIP_TRY(launch_gemm_f32(epi, s));
    if (rec) rec->end();
    return RAVEL_OK;
  }
  if ((K % 8) || (lda % 8) || (ldb % 8)) return fail(RAVEL_E_SHAPE, std::string(name) + ": K and strides must be multiples of 8");
  const GemmPlan p = plan_gemm(M, N, K, epi.mode == EPI_GEGLU);
  epi.ksplit = epi.m_rows ? 1 : p.ksplit;  // device row count: whole K per block
  epi.kchunk = epi.m_rows ? K : p.kchunk;
  epi.partial = b->gpart;
  epi.counters = b->gcnt;
  if (p.part_elems > b->gpart_elems || p.tiles > b->gcnt_n)
    return fail(RAVEL_E_STATE, std::string(name) + ": GEMM workspace too small");
  if (epi.m_rows && p.skinny) return fail(RAVEL_E_STATE, std::string(name) + ": device row count needs a tiled GEMM");
  if (rec) {
    static const char* tn[] = {"64x64", "128x128", "64x128", "128x64", "32x64", "256x128", "128x256", "256x256"};
    char full[48];
    if (epi.m_rows)  // rows known on the device only: no byte / flop figures
      snprintf(full, sizeof full, "gemm_rows:%s", name);
    else if (p.skinny && p.wholek)
      snprintf(full, sizeof full, "gemm_wholek<%d>:%s", (M + 15) / 16, name);
    else if (p.skinny && p.regstream)
      snprintf(full, sizeof full, "gemm_regstream<%d>:%s", (M + 15) / 16, name);
    else if (p.skinny)
      snprintf(full, sizeof full, "gemm_stream<%d,%d>:%s", (M + 15) / 16, p.kchunk, name);
    else
      snprintf(full, sizeof full, "gemm%s:%s", tn[p.tile], name);
    rec->begin(full, epi.m_rows ? 0.0 : bytes, epi.m_rows ? 0.0 : flops);
  }
  if (p.skinny) {
    if (p.wholek)
      HIP_TRY(launch_gemm_wholek(epi, s));
    else if (p.regstream)
      HIP_TRY(launch_gemm_regstream(epi, s));
    else
      HIP_TRY(launch_gemm_skinny(epi, p.nfr, s));
    if (rec) rec->end();
    return RAVEL_OK;
  }
  HIP_TRY(launch_gemm_bf16(epi, p.tile, s));
  if (rec) rec->end();
  return RAVEL_OK;
}

GemmArgs epi_args(int mode) {
  GemmArgs a;
  memset(&a, 0, sizeof a);
  a.mode = mode;
  a.ksplit = 1;
  return a;
}

template <typename T>
ravel_status run_attn(ravel_buffer* b, hipStream_t s, KernelRecorder* rec, const char* name, AttnArgs a) {
  ravel_model* m = b->m;
  const ravel_config& c = m->cfg;
  a.B = b->B;
  a.nq = c.n_q_heads;
  a.nkv = c.n_kv_heads;
  a.hd = c.head_dim;
  a.scale = 1.0f / sqrtf((float)c.head_dim);
  const int nkeys = a.P + a.S;
  if (m->bf16 && a.S > 0 && b->attn_nsplit > 1) {
    a.nsplit = b->attn_nsplit;
    a.keys_per_split = b->attn_kps;
  } else {
    a.nsplit = 1;
    a.keys_per_split = ((nkeys + 31) / 32) * 32;
  }
  a.part_o = b->apart_o;
  a.part_ml = b->apart_ml;
  a.counters = b->acnt;
  const double elt = (double)m->elt;
  const double bytes = (double)b->B * (a.Hq * (double)c.n_q_heads * c.head_dim * 2 * elt +
                                       (double)nkeys * c.n_kv_heads * c.head_dim * 2 * elt);
  const double flops = 4.0 * b->B * c.n_q_heads * (double)a.Hq * nkeys * c.head_dim;
  if (rec) rec->begin(name, bytes, flops);
  if (m->bf16)
    HIP_TRY(launch_attn_bf16(a, s));
  else
    HIP_TRY(launch_attn_f32(a, s));
  if (rec) rec->end();
  return RAVEL_OK;
}

#define REC_BEGIN(nm, by, fl) \
  if (rec) rec->begin(nm, by, fl)
#define REC_END() \
  if (rec) rec->end()

constexpr int kMaxFullSteps = 1024;  // Euler steps of one full-horizon chunk

// What one expert pass reads: the rolling ring (its slots at the buffer's flow-time
// profile, context age t - t_obs), or a full-horizon chunk whose slots share one
// flow time (row tau_row of the table ctau) at context age 0.
struct PassIn {
  const float* X = nullptr;     // [B, H, D] chunk in logical order; NULL: the ring
  const float* ctau = nullptr;  // conditioning table; NULL: the model's rolling table
  int tau_row = -1;             // every slot uses this table row; -1: slot i uses row i
  const int64_t* ages = nullptr;  // [B] context age per env (device) instead of t - t_obs / 0
  int tau_den = 0;                // with tau_row >= 0: that row's flow time is (tau_row + 1) / tau_den
  bool lead_bias = true;          // add delta_0 to the offset (inference); training uses p / H alone
};

// DynamicVLA-style offset form (App. A.1) on the encoded actions x = W_in a + b_in:
// x = W_a2 silu(W_a1 [x ; emb(tau) ; delta] + b_a1) + b_a2 (the action-time MLP), then
// x += tanh(beta) W_r2 silu(W_r1 [x ; emb(delta)] + b_r1) (the gated residual adapter).
template <typename T>
ravel_status enqueue_offset_adapter(ravel_buffer* b, hipStream_t s, KernelRecorder* rec, const PassIn& pin) {
  ravel_model* m = b->m;
  const ravel_config& c = m->cfg;
  const int B = b->B, H = c.horizon, w = c.width, BH = B * H, Kz = m->at_kz, r = w / 4;
  const double elt = (double)m->elt;
  REC_BEGIN("offset_rows", (double)BH * w * 4 + (double)BH * Kz * elt, 0.0);
  HIP_TRY(launch_offset_rows<T>(0, b->x, b->dval, B, H, w, pin.tau_row, pin.tau_den, (T*)b->tz, Kz, s));
  REC_END();
  GemmArgs e1 = epi_args(EPI_SILU_T);
  e1.bias = m->at_b1;
  e1.out_t = b->th;
  e1.ldo_t = w;
  RV_TRY(run_gemm<T>(b, s, rec, "action_time1", b->tz, Kz, m->at_w1, Kz, BH, w, Kz, e1));
  GemmArgs e2 = epi_args(EPI_F32);
  e2.bias = m->at_b2;
  e2.out_f = b->x;
  e2.ldo_f = w;
  RV_TRY(run_gemm<T>(b, s, rec, "action_time2", b->th, w, m->at_w2, w, BH, w, w, e2));
  REC_BEGIN("offset_rows", (double)BH * w * 4 + (double)BH * 2 * w * elt, 0.0);
  HIP_TRY(launch_offset_rows<T>(1, b->x, b->dval, B, H, w, -1, 0, (T*)b->tz, Kz, s));
  REC_END();
  GemmArgs e3 = epi_args(EPI_SILU_T);
  e3.bias = m->ta_b1;
  e3.out_t = b->th;
  e3.ldo_t = r;
  RV_TRY(run_gemm<T>(b, s, rec, "offset_adapter1", b->tz, Kz, m->ta_w1, 2 * w, BH, r, 2 * w, e3));
  GemmArgs e4 = epi_args(EPI_RESID_TANH);
  e4.gate_scalar = m->ta_alpha;
  e4.out_f = b->x;
  e4.ldo_f = w;
  RV_TRY(run_gemm<T>(b, s, rec, "offset_adapter2", b->th, r, m->ta_w2, r, BH, w, r, e4));
  return RAVEL_OK;
}

template <typename T>
ravel_status enqueue_transformer(ravel_buffer* b, const void* fop, hipStream_t s, KernelRecorder* rec,
                                 const PassIn& pin) {
  ravel_model* m = b->m;
  const ravel_config& c = m->cfg;
  const int B = b->B, H = c.horizon, w = c.width, D = c.action_dim;
  const int BH = B * H;
  const int qd = c.n_q_heads * c.head_dim, kvd = c.n_kv_heads * c.head_dim;
  const int qkvd = qd + 2 * kvd;
  const int F = c.mlp_dim;
  const double elt = (double)m->elt;

  // 1. offset conditioning: delta_e = p/H + delta_0, d = W_d2 silu(W_d1 delta + b_d1) + b_d2,
  //    cond[e,i] = silu(c_tau(i) + d); or, with the offset concatenated to the inputs (or
  //    fed to the action-time MLP and adapter), cond[e,i] = silu(c_tau(i)) and delta_e
  //    goes to the action encoder
  const bool concat = c.offset_mode == RAVEL_OFFSET_CONCAT;
  const bool no_mlp = c.offset_mode != RAVEL_OFFSET_MLP;
  const float dbias = pin.lead_bias ? c.delta_bias : 0.f;
  if (no_mlp) {
    REC_BEGIN("offset_value", (double)B * 12, 0.0);
    HIP_TRY(launch_offset_value(pin.X ? nullptr : b->t, b->t_obs, pin.ages, B, H, dbias, b->dval, s));
    REC_END();
  } else {
    REC_BEGIN("delta_hidden", (double)B * w * (8 + elt), (double)B * w * 4);
    HIP_TRY(launch_delta_hidden<T>(pin.X ? nullptr : b->t, b->t_obs, pin.ages, B, H, dbias, m->d_w1, m->d_b1, w,
                                   (T*)b->h1, s));
    REC_END();
  }
  // Envs with equal t_obs have equal delta, so equal cond rows and modulation
  // rows: cond is written once per group (compacted) and the modulation GEMM
  // runs on the groups' rows only.
  const int* rowmap = b->cgroups ? b->crowmap : nullptr;
  if (b->cgroups) {
    REC_BEGIN("cond_groups", (double)B * 8 + (double)BH * 4, 0.0);
    // equal context ages give equal offsets (the shared t makes equal t_obs equal ages)
    HIP_TRY(launch_cond_groups(pin.ages ? pin.ages : b->t_obs, B, H, b->cgrp, b->crowmap, b->crows, s));
    REC_END();
  }
  if (!no_mlp) {
    GemmArgs e = epi_args(EPI_F32);
    e.bias = m->d_b2;
    e.out_f = b->dvec;
    e.ldo_f = w;
    RV_TRY(run_gemm<T>(b, s, rec, "cond", b->h1, w, m->d_w2, w, B, w, w, e));
  }
  REC_BEGIN("cond_expand", (double)B * w * 4 + (double)H * w * 4 + (double)BH * w * elt, (double)BH * w * 4);
  HIP_TRY(launch_cond_expand<T>(no_mlp ? nullptr : b->dvec, B, H, w, pin.ctau ? pin.ctau : m->ctau, pin.tau_row,
                                b->cgroups ? b->cgrp : nullptr, (T*)b->cond, s));
  REC_END();
  // 2. input projection of the buffer in logical order
  REC_BEGIN("in_proj", (double)BH * (D + w) * 4, 2.0 * BH * w * D);
  HIP_TRY(launch_in_proj(pin.X ? pin.X : b->X, pin.X ? nullptr : b->t, B, H, D, m->in_wT, m->in_b, w, b->x,
                         InProjNorm{}, concat ? b->dval : nullptr, s));
  REC_END();
  if (c.offset_mode == RAVEL_OFFSET_ADAPTER) RV_TRY(enqueue_offset_adapter<T>(b, s, rec, pin));
  // FOP adapter keys/values of every adapter layer at once
  if (m->n_ad > 0) {
    GemmArgs e = epi_args(EPI_T);
    e.out_t = b->kva;
    e.ldo_t = m->n_ad * 2 * kvd;
    RV_TRY(run_gemm<T>(b, s, rec, "fop_kv", fop, w, m->kva_w, w, B * c.n_fop, m->n_ad * 2 * kvd, w, e));
  }
  const size_t ctx_layer = (size_t)c.prefix_len * kvd;
  const int ldm = b->mod_ld;
  if (b->mod_all) {
    // modulation chunks (s1, b1, g1, s2, b2, g2) of every layer and (s_f, b_f) at once
    GemmArgs e = epi_args(EPI_F32);
    e.bias = m->mod_all_b;
    e.out_f = b->mod;
    e.ldo_f = ldm;
    e.m_rows = b->cgroups ? b->crows : nullptr;
    RV_TRY(run_gemm<T>(b, s, rec, "mod_all", b->cond, w, m->mod_all_w, w, BH, ldm, w, e));
  }
  for (int l = 0; l < c.layers; ++l) {
    const LayerW& L = m->layers[l];
    const float* mod = b->mod_all ? b->mod + (size_t)l * 6 * w : b->mod;
    if (!b->mod_all) {
      GemmArgs e = epi_args(EPI_F32);
      e.bias = L.mod_b;
      e.out_f = b->mod;
      e.ldo_f = ldm;
      RV_TRY(run_gemm<T>(b, s, rec, "mod", b->cond, w, L.mod_w, w, BH, 6 * w, w, e));
    }
    REC_BEGIN("adarms", (double)BH * w * (12 + elt), (double)BH * w * 5);
    HIP_TRY(launch_adarms<T>(b->x, w, BH, w, mod, mod + w, ldm, 0, rowmap, c.rms_eps, (T*)b->y, w, s));
    REC_END();
    {
      GemmArgs e = epi_args(EPI_T);
      e.out_t = b->qkv;
      e.ldo_t = qkvd;
      RV_TRY(run_gemm<T>(b, s, rec, "qkv", b->y, w, L.qkv_w, w, BH, qkvd, w, e));
    }
    if (m->rope_cs) {
      REC_BEGIN("rope", (double)BH * (qd + kvd) * 2 * elt + (double)H * c.head_dim * 4, 0.0);
      HIP_TRY(launch_rope<T>((T*)b->qkv, qkvd, BH, H, c.n_q_heads, c.n_kv_heads, c.head_dim, m->rope_cs, s));
      REC_END();
    }
    {
      AttnArgs a;
      memset(&a, 0, sizeof a);
      a.q = b->qkv;
      a.ldq = qkvd;
      a.Hq = H;
      a.pk = (const char*)b->ctx_k + l * ctx_layer * m->elt;
      a.pv = (const char*)b->ctx_v + l * ctx_layer * m->elt;
      a.p_env_stride = (long long)b->ctx_elems;
      a.p_slot_stride = (long long)b->ctx_elems * B;
      a.slot = b->slot;
      a.P = c.prefix_len;
      a.p_ld = kvd;
      a.sk = (const char*)b->qkv + (size_t)qd * m->elt;
      a.sv = (const char*)b->qkv + (size_t)(qd + kvd) * m->elt;
      a.S = H;
      a.s_ld = qkvd;
      a.out = b->att;
      a.ldo = qd;
      RV_TRY(run_attn<T>(b, s, rec, "attn", a));
    }
    {
      GemmArgs e = epi_args(EPI_RESID);
      e.out_f = b->x;
      e.ldo_f = w;
      e.gate = mod + 2 * w;
      e.ldg = ldm;
      e.gate_rows = rowmap;
      RV_TRY(run_gemm<T>(b, s, rec, "o", b->att, qd, L.o_w, qd, BH, w, qd, e));
    }
    if (L.adapter >= 0 && fop) {
      REC_BEGIN("adarms", (double)BH * w * (8 + elt), (double)BH * w * 4);
      HIP_TRY(launch_adarms<T>(b->x, w, BH, w, L.gamma, nullptr, 0, 1, nullptr, c.rms_eps, (T*)b->y, w, s));
      REC_END();
      {
        GemmArgs e = epi_args(EPI_T);
        e.out_t = b->qa;
        e.ldo_t = qd;
        RV_TRY(run_gemm<T>(b, s, rec, "fop_q", b->y, w, L.qa_w, w, BH, qd, w, e));
      }
      {
        AttnArgs a;
        memset(&a, 0, sizeof a);
        const int ld = m->n_ad * 2 * kvd;
        a.q = b->qa;
        a.ldq = qd;
        a.Hq = H;
        a.pk = (const char*)b->kva + (size_t)L.adapter * 2 * kvd * m->elt;
        a.pv = (const char*)b->kva + (size_t)(L.adapter * 2 * kvd + kvd) * m->elt;
        a.p_env_stride = (long long)c.n_fop * ld;
        a.p_slot_stride = 0;
        a.slot = nullptr;
        a.P = c.n_fop;
        a.p_ld = ld;
        a.sk = nullptr;
        a.sv = nullptr;
        a.S = 0;
        a.s_ld = 0;
        a.out = b->att;
        a.ldo = qd;
        RV_TRY(run_attn<T>(b, s, rec, "fop_attn", a));
      }
      {
        GemmArgs e = epi_args(EPI_RESID_TANH);
        e.out_f = b->x;
        e.ldo_f = w;
        e.gate_scalar = L.alpha;
        RV_TRY(run_gemm<T>(b, s, rec, "fop_o", b->att, qd, L.oa_w, qd, BH, w, qd, e));
      }
    }
    REC_BEGIN("adarms", (double)BH * w * (12 + elt), (double)BH * w * 5);
    HIP_TRY(launch_adarms<T>(b->x, w, BH, w, mod + 3 * w, mod + 4 * w, ldm, 0, rowmap, c.rms_eps, (T*)b->y, w, s));
    REC_END();
    {
      GemmArgs e = epi_args(EPI_GEGLU);
      e.out_t = b->u;
      e.ldo_t = F;
      RV_TRY(run_gemm<T>(b, s, rec, "gate_up", b->y, w, L.gu_w, w, BH, 2 * F, w, e));
    }
    {
      GemmArgs e = epi_args(EPI_RESID);
      e.out_f = b->x;
      e.ldo_f = w;
      e.gate = mod + 5 * w;
      e.ldg = ldm;
      e.gate_rows = rowmap;
      RV_TRY(run_gemm<T>(b, s, rec, "down", b->u, F, L.down_w, F, BH, w, F, e));
    }
  }
  // final adaptive norm and output head
  const float* fmod = b->mod_all ? b->mod + (size_t)c.layers * 6 * w : b->fmod;
  const int ldf = b->mod_all ? ldm : 2 * w;
  if (!b->mod_all) {
    GemmArgs e = epi_args(EPI_F32);
    e.bias = m->fmod_b;
    e.out_f = b->fmod;
    e.ldo_f = 2 * w;
    RV_TRY(run_gemm<T>(b, s, rec, "final_mod", b->cond, w, m->fmod_w, w, BH, 2 * w, w, e));
  }
  REC_BEGIN("adarms", (double)BH * w * (12 + elt), (double)BH * w * 5);
  HIP_TRY(launch_adarms<T>(b->x, w, BH, w, fmod, fmod + w, ldf, 0, rowmap, c.rms_eps, (T*)b->y, w, s));
  REC_END();
  {
    GemmArgs e = epi_args(EPI_F32);
    e.bias = m->out_b;
    e.out_f = b->v;
    e.ldo_f = D;
    RV_TRY(run_gemm<T>(b, s, rec, "out", b->y, w, m->out_w, w, BH, D, w, e));
  }
  return RAVEL_OK;
}

ravel_status enqueue_step(ravel_buffer* b, const void* fop, const float* state, float* action, hipStream_t s,
                          KernelRecorder* rec) {
  ravel_model* m = b->m;
  const ravel_config& c = m->cfg;
  const int B = b->B, H = c.horizon, D = c.action_dim;
  if (state) {
    REC_BEGIN("relative_shift", (double)B * H * D * 8 + (double)B * D * 8, (double)B * H * D * 3);
    HIP_TRY(launch_relative_shift(b->X, b->t, B, H, D, b->rel_mask, state, b->s_prev, b->has_prev, s));
    REC_END();
  }
  if (c.model_kind == RAVEL_TRANSFORMER) {
    if (m->bf16)
      RV_TRY(enqueue_transformer<bf16_t>(b, fop, s, rec, PassIn{}));
    else
      RV_TRY(enqueue_transformer<float>(b, fop, s, rec, PassIn{}));
  } else {
    REC_BEGIN("analytic_velocity", (double)B * H * D * 8, (double)B * H * D * 2);
    HIP_TRY(launch_analytic_velocity(c.model_kind, b->X, b->t, B, H, D, m->analytic, 0.f, state, b->rel_mask, b->v,
                                     s));
    REC_END();
  }
  REC_BEGIN("euler_release", (double)B * H * D * 12 + (double)B * D * 4, (double)B * H * D * 2);
  HIP_TRY(launch_euler_release(b->X, b->v, b->t, B, H, D, b->seed, action, b->ticket, state, b->rel_mask, nullptr, nullptr, s));
  REC_END();
  return RAVEL_OK;
}

// Apply ready context publishes on the step stream (caller holds the mutex).
ravel_status apply_publishes(ravel_buffer* b, hipStream_t s) {
  PublishBatch pb;
  memset(&pb, 0, sizeof pb);
  for (int e = 0; e < b->B; ++e) {
    PendingCtx& p = b->pending[e];
    if (!p.valid) continue;
    if (b->sync_ctx) {
      HIP_TRY(hipStreamWaitEvent(s, p.ready, 0));
    } else {
      const hipError_t q = hipEventQuery(p.ready);
      if (q == hipErrorNotReady) continue;
      if (q != hipSuccess) return fail(RAVEL_E_HIP, std::string("hipEventQuery: ") + hipGetErrorString(q));
    }
    // the slot that stops being read: free once the steps enqueued so far are done
    HIP_TRY(hipEventRecord(b->retire[e], s));
    b->retire_valid[e] = 1;
    const int ns = b->has_ctx[e] ? 1 - b->active[e] : b->active[e] ^ 1;
    b->active[e] = ns;
    b->has_ctx[e] = 1;
    b->tobs_host[e] = p.t_obs;
    b->log.push_back({(int64_t)e, b->t_host, p.t_obs});
    p.valid = false;
    pb.env[pb.n] = e;
    pb.new_slot[pb.n] = ns;
    pb.tobs[pb.n] = p.t_obs;
    if (++pb.n == 32) {
      HIP_TRY(launch_publish(pb, b->slot, b->t_obs, s));
      pb.n = 0;
    }
  }
  if (pb.n) HIP_TRY(launch_publish(pb, b->slot, b->t_obs, s));
  return RAVEL_OK;
}

ravel_status acquire_locked(ravel_buffer* b, int env, void** k, void** v, hipStream_t producer) {
  ravel_model* m = b->m;
  b->pending[env].valid = false;  // a not-yet-applied publish of this env is superseded
  const int inactive = b->has_ctx[env] ? 1 - b->active[env] : (b->active[env] ^ 1);
  if (b->retire_valid[env]) HIP_TRY(hipStreamWaitEvent(producer, b->retire[env], 0));
  const size_t off = ((size_t)inactive * b->B + env) * b->ctx_elems * m->elt;
  *k = (char*)b->ctx_k + off;
  *v = (char*)b->ctx_v + off;
  return RAVEL_OK;
}


// ---------------------------------------------------------------------------
// Persistent few-row path: phase list of the transformer layers
// ---------------------------------------------------------------------------
bool persistent_eligible(const ravel_buffer* b) {
  const ravel_model* m = b->m;
  const ravel_config& c = m->cfg;
  if (!m->bf16 || c.model_kind != RAVEL_TRANSFORMER || !b->mod_all) return false;
  const int BH = b->B * c.horizon, hd = c.head_dim;
  const int qd = c.n_q_heads * hd, kvd = c.n_kv_heads * hd;
  if (BH > 64 || b->B > 64) return false;
  if (hd != 32 && hd != 64 && hd != 128 && hd != 256) return false;
  // 64-column output tiles everywhere but the output head; K ranges of 256 or
  // 512 with at most kMaxKSplit of them
  if (c.width % 64 || qd % 64 || (qd + 2 * kvd) % 64 || c.mlp_dim % 32) return false;
  for (int K : {c.width, qd, c.mlp_dim})
    if (K % 8 || (K + 511) / 512 > kMaxKSplit) return false;
  if (c.width > 4096) return false;  // row sums of squares: at most 64 tiles
  if (c.n_fop > attn_keys_per_split_max(hd)) return false;
  const int kmax = attn_keys_per_split_max(hd);
  if ((c.prefix_len + kmax - 1) / kmax + (c.horizon + kmax - 1) / kmax > kMaxAttnSplit) return false;
  return true;
}

template <class T>
ravel_status palloc(ravel_buffer* b, T** p, size_t bytes, bool zero) {
  void* q = nullptr;
  HIP_TRY(hipMalloc(&q, std::max<size_t>(bytes, 256)));
  b->pallocs.push_back(q);
  if (zero) HIP_TRY(hipMemset(q, 0, std::max<size_t>(bytes, 256)));
  *p = (T*)q;
  return RAVEL_OK;
}

// Phase list of the persistent kernel (see persistent.hip), with its workspaces.
ravel_status build_persistent(ravel_buffer* b) {
  ravel_model* m = b->m;
  const ravel_config& c = m->cfg;
  const int B = b->B, H = c.horizon, w = c.width, D = c.action_dim, BH = B * H, F = c.mlp_dim, hd = c.head_dim;
  const int qd = c.n_q_heads * hd, kvd = c.n_kv_heads * hd, qkvd = qd + 2 * kvd;
  const int ldm = b->mod_ld;
  int mt = (BH + 15) / 16;
  if (mt == 3) mt = 4;
  b->pmt = mt;
  b->pblocks = std::min(persistent_max_blocks(mt, hd), 256);
  if (b->pblocks < 64) return fail(RAVEL_E_STATE, "persistent kernel does not fit");
  auto tiles = [](int n) { return (n + 63) / 64; };
  RV_TRY(palloc(b, &b->pbar, kBarrierWords * 4, true));
  RV_TRY(palloc(b, &b->perr, 64, true));
  RV_TRY(palloc(b, &b->sumsq[0], (size_t)(w / 64) * 64 * 4, true));
  RV_TRY(palloc(b, &b->pnorm, (size_t)64 * w * 2, true));
  // bf16 copies of the norm shifts: chunk 2l (attention) and 2l + 1 (MLP) of
  // layer l, 2L the final norm; in the modulation rows they sit 3w apart
  // starting at column w.  Like every p of a norm, they are stored in 32-column
  // tiles [w/32][64 rows][32], so that a GEMM item's 16-row fragment loads are
  // 1 KB contiguous (about 1.5x the rate of 64-byte pieces of 16 rows).
  const int nshift = 2 * c.layers + 1;
  RV_TRY(palloc(b, &b->pshift, (size_t)nshift * 64 * w * 2, true));
  // Every activation a phase writes gets buffers of its own (written once per
  // launch, read with plain loads by the phases after it): one arena, bumped in
  // phase order.  Row sums of squares take one 128-byte line per (tile, row).
  const size_t sq_bytes = (size_t)(w / 64) * 64 * 32 * 4;
  const size_t resid_bytes = align_up((size_t)BH * w * 4, 256) + align_up((size_t)64 * w * 2, 256) + sq_bytes;
  const bool rope = m->rope_cs != nullptr;
  size_t act_bytes = 0;
  for (int l = 0; l < c.layers; ++l) {
    const bool ad = m->layers[l].adapter >= 0;
    act_bytes += align_up((size_t)BH * qkvd * 2, 256) * (rope ? 2 : 1);                   // QKV (+ rotated)
    act_bytes += align_up((size_t)BH * qd * 2, 256);                                       // attention output
    act_bytes += resid_bytes * (ad ? 3 : 2);                                               // x, p, sums per update
    if (ad) act_bytes += align_up((size_t)BH * qd * 2, 256) * 2;  // adapter queries (+ cross-attention output)
    act_bytes += align_up((size_t)(F / 32) * 2048 * 2, 256);                               // MLP hidden, 32-col tiles
  }
  char* act = nullptr;
  RV_TRY(palloc(b, &act, act_bytes, true));
  size_t act_off = 0;
  auto fresh = [&](size_t bytes) -> void* {
    void* q = act + act_off;
    act_off += align_up(bytes, 256);
    return q;
  };
  // the current residual, the next norm's p and row sums (the input projection
  // writes the first ones before the launch, sums unpadded)
  const float* cur_x = b->x;
  const bf16_t* cur_p = (const bf16_t*)b->pnorm;
  const float* cur_sq = b->sumsq[0];
  int cur_sq_ld = 1;
  const bf16_t* pshift = b->pshift;
  auto shift_of = [&](int chunk) -> const bf16_t* { return pshift + (size_t)chunk * 64 * w; };
  size_t part = 0;
  std::vector<Phase>& P = b->phases;
  P.clear();
  b->pnames.clear();
  auto push = [&](const Phase& ph, const char* name) {
    P.push_back(ph);
    b->pnames.push_back(name);
  };
  bool whole_k = true;
  if (const char* ev = getenv("RAVEL_NO_WHOLE_K")) whole_k = atoi(ev) == 0;
  auto gemm = [&](const void* A, int lda, const bf16_t* shift, bool norm, const void* W, int N, int K, int e_mode) {
    Phase ph;
    memset(&ph, 0, sizeof ph);
    ph.type = PH_GEMM;
    PGemm& g = ph.g;
    g.a_mode = norm ? PA_NORM : PA_BF16;
    g.A = (const bf16_t*)A;
    g.lda = lda;
    g.shift = shift;
    g.ld_shift = w;
    // p and the shift copies of a norm are stored in 32-column tiles
    g.sh_t32 = norm ? 1 : 0;
    g.a_t32 = norm ? 1 : 0;
    g.sumsq_in = cur_sq;
    g.sq_in_ld = cur_sq_ld;
    g.eps = c.rms_eps;
    g.W = (const bf16_t*)W;
    g.ldw = K;
    g.M = BH;
    g.N = N;
    g.K = K;
    const int ks1 = (K + 255) / 256;
    g.kw = (ks1 <= kMaxKSplit && tiles(N) * ks1 <= b->pblocks) ? 1 : 2;
    if ((K + 256 * g.kw - 1) / (256 * g.kw) > kMaxKSplit) g.kw = 0;  // rejected below
    g.ksplit = (K + 256 * g.kw - 1) / (256 * g.kw);
    g.e_mode = e_mode;
    g.counters = nullptr;  // patched below
    // a K that would be split over blocks and fits four waves' quarters of at most
    // 256: whole-K items of 16 columns (a gate block and its up block for GeGLU)
    const int wk = e_mode == PE_GEGLU ? 2 : 1;
    if (whole_k && norm && g.ksplit > 1 && K % 128 == 0 && K <= 1024 && N % (16 * wk) == 0 &&
        (e_mode == PE_BF16 || e_mode == PE_F32 || e_mode == PE_GEGLU)) {
      g.wk = wk;
      g.kw = 1;
      g.ksplit = 1;
      ph.items = N / (16 * wk);
      return ph;
    }
    ph.items = tiles(N) * g.ksplit;
    g.coop = g.ksplit > 1 && ph.items <= b->pblocks;
    part = std::max(part, (size_t)g.ksplit * tiles(N) * mt * 4 * 64 * 4);
    return ph;
  };
  auto resid = [&](Phase& ph, const float* gate, const float* gate_scalar, int ns_mode, const float* ns) {
    PGemm& g = ph.g;
    g.x_in = cur_x;
    g.out_f = (float*)fresh((size_t)BH * w * 4);
    g.ldof = w;
    g.gate = gate;
    g.ldg = ldm;
    g.gate_scalar = gate_scalar;
    g.ns_mode = ns_mode;
    g.ns = ns;
    g.ldns = ldm;
    g.p_out = (bf16_t*)fresh((size_t)64 * w * 2);
    g.ldp = w;
    g.p_t32 = 1;
    g.sumsq_out = (float*)fresh(sq_bytes);
    g.sq_out_ld = 32;
    cur_x = g.out_f;
    cur_p = g.p_out;
    cur_sq = g.sumsq_out;
    cur_sq_ld = 32;
  };
  // the input projection writes the first norm's p and row sums of squares
  // (b->sumsq[0]) and the bf16 shifts before the launch
  int max_attn_parts = 1;
  auto attn_phase = [&](AttnArgs a) {
    Phase ph;
    memset(&ph, 0, sizeof ph);
    ph.type = PH_ATTN;
    a.B = B;
    a.nq = c.n_q_heads;
    a.nkv = c.n_kv_heads;
    a.hd = hd;
    a.scale = 1.0f / sqrtf((float)hd);
    // splits of at most kmax keys (a multiple of 32) over the prefix, then over
    // the self keys: no split holds both kinds
    const int kmax = attn_keys_per_split_max(hd);
    const int np = std::max((a.P + kmax - 1) / kmax, 1);
    a.keys_per_split = std::min(kmax, (((a.P + np - 1) / np + 31) / 32) * 32);
    a.keys_per_split = std::max(a.keys_per_split, std::min(kmax, ((a.S + 31) / 32) * 32));
    a.nsplit = (a.P + a.keys_per_split - 1) / a.keys_per_split + (a.S + a.keys_per_split - 1) / a.keys_per_split;
    ph.items = B * c.n_q_heads * a.nsplit;
    a.coop = a.nsplit > 1 && ph.items <= b->pblocks;
    ph.at = a;
    max_attn_parts = std::max(max_attn_parts, B * c.n_q_heads * a.nsplit);
    return ph;
  };
  const size_t ctx_layer = (size_t)c.prefix_len * kvd;
  bool xattn_fused = B == 1 && hd == 256 && c.n_fop >= 1 && c.n_fop <= 16 && c.n_q_heads % c.n_kv_heads == 0;
  if (const char* ev = getenv("RAVEL_NO_FUSED_XATTN")) xattn_fused = xattn_fused && atoi(ev) == 0;
  // an attention output is written in (query, head) segments of hd bf16 values by
  // each head's merge: whole 128-byte lines only when hd >= 64
  const int att_coh = hd < 64 ? 1 : 0;
  // outputs of whole-K items are written in 16-column pieces (several writers per
  // 128-byte line): their readers use device-coherent loads
  bool qkv_pieces = false, qa_pieces = false, u_pieces = false;
  // per layer: its first phase and its gate/up phase (the side work of layer l, the
  // modulation of layer l + 1 or of the final norm, runs in the phases between)
  std::vector<int> layer_first(c.layers), layer_gu(c.layers);
  for (int l = 0; l < c.layers; ++l) {
    const LayerW& L = m->layers[l];
    layer_first[l] = (int)P.size();
    const float* mod = b->mod + (size_t)l * 6 * w;
    const float* next_scale = b->mod + (size_t)(l + 1) * 6 * w;  // next layer's (or the final) chunk 0
    bf16_t* qkv = (bf16_t*)fresh((size_t)BH * qkvd * 2);
    {
      Phase ph = gemm(cur_p, w, shift_of(2 * l), true, L.qkv_w, qkvd, w, PE_BF16);
      ph.g.out_t = qkv;
      ph.g.ldo = qkvd;
      qkv_pieces = ph.g.wk != 0;
      push(ph, "qkv");
    }
    // queries and keys as attention reads them: rotated into a buffer of their own
    const bf16_t* qk = qkv;
    if (rope) {
      bf16_t* rot = (bf16_t*)fresh((size_t)BH * qkvd * 2);
      Phase ph;
      memset(&ph, 0, sizeof ph);
      ph.type = PH_ROPE;
      ph.items = BH;
      ph.r.qkv = qkv;
      ph.r.out = rot;
      ph.r.ld = qkvd;
      ph.r.H = H;
      ph.r.nh = c.n_q_heads + c.n_kv_heads;
      ph.r.hd = hd;
      ph.r.cs = m->rope_cs;
      ph.r.coh = qkv_pieces ? 1 : 0;
      push(ph, "rope");
      qk = rot;
    }
    bf16_t* att = (bf16_t*)fresh((size_t)BH * qd * 2);
    {
      AttnArgs a;
      memset(&a, 0, sizeof a);
      a.q = qk;
      a.ldq = qkvd;
      a.Hq = H;
      a.pk = (const char*)b->ctx_k + l * ctx_layer * m->elt;
      a.pv = (const char*)b->ctx_v + l * ctx_layer * m->elt;
      a.p_env_stride = (long long)b->ctx_elems;
      a.p_slot_stride = (long long)b->ctx_elems * B;
      a.slot = b->slot;
      a.P = c.prefix_len;
      a.p_ld = kvd;
      a.sk = (const char*)qk + (size_t)qd * m->elt;
      a.sv = (const char*)qkv + (size_t)(qd + kvd) * m->elt;
      a.S = H;
      a.s_ld = qkvd;
      a.out = att;
      a.ldo = qd;
      a.coh = qkv_pieces ? 1 : 0;
      push(attn_phase(a), "self_attn");
    }
    {
      Phase ph = gemm(att, qd, nullptr, false, L.o_w, w, qd, PE_RESID);
      ph.g.a_coh = att_coh;
      if (L.adapter >= 0)
        resid(ph, mod + 2 * w, nullptr, NS_COL, L.gamma);
      else
        resid(ph, mod + 2 * w, nullptr, NS_ROW, mod + 3 * w);
      push(ph, "o_proj");
    }
    if (L.adapter >= 0) {
      bf16_t* qa = (bf16_t*)fresh((size_t)BH * qd * 2);
      {
        Phase ph = gemm(cur_p, w, nullptr, true, L.qa_w, qd, w, PE_BF16);
        ph.g.out_t = qa;
        ph.g.ldo = qd;
        qa_pieces = ph.g.wk != 0;
        push(ph, "q_adapter");
      }
      // one env, heads of 256 dims, at most 16 FOP tokens: the output projection's
      // items compute their head's cross-attention themselves (no attention phase)
      const int ld = m->n_ad * 2 * kvd;
      Phase fused = gemm(qa, qd, nullptr, false, L.oa_w, w, qd, PE_RESID);
      if (xattn_fused && fused.g.kw == 1) {
        resid(fused, nullptr, L.alpha, NS_ROW, mod + 3 * w);
        PGemm& g = fused.g;
        g.a_mode = PA_XATTN;
        g.xk = (const bf16_t*)b->kva + (size_t)L.adapter * 2 * kvd;
        g.xv = g.xk + kvd;
        g.x_ld = ld;
        g.x_nf = c.n_fop;
        g.x_group = c.n_q_heads / c.n_kv_heads;
        g.x_scale = 1.0f / sqrtf((float)hd);
        g.a_coh = qa_pieces ? 1 : 0;
        push(fused, "o_adapter");
      } else {
        bf16_t* xatt = (bf16_t*)fresh((size_t)BH * qd * 2);
        AttnArgs a;
        memset(&a, 0, sizeof a);
        a.q = qa;
        a.ldq = qd;
        a.Hq = H;
        a.pk = (const char*)b->kva + (size_t)L.adapter * 2 * kvd * m->elt;
        a.pv = (const char*)b->kva + (size_t)(L.adapter * 2 * kvd + kvd) * m->elt;
        a.p_env_stride = (long long)c.n_fop * ld;
        a.P = c.n_fop;
        a.p_ld = ld;
        a.S = 0;
        a.out = xatt;
        a.ldo = qd;
        a.coh = qa_pieces ? 1 : 0;
        push(attn_phase(a), "cross_attn");
        Phase ph = gemm(xatt, qd, nullptr, false, L.oa_w, w, qd, PE_RESID);
        ph.g.a_coh = att_coh;
        resid(ph, nullptr, L.alpha, NS_ROW, mod + 3 * w);
        push(ph, "o_adapter");
      }
    }
    bf16_t* u = (bf16_t*)fresh((size_t)(F / 32) * 2048 * 2);
    {
      Phase ph = gemm(cur_p, w, shift_of(2 * l + 1), true, L.gu_w, 2 * F, w, PE_GEGLU);
      ph.g.out_t = u;
      ph.g.ldo = F;
      ph.g.out_t32 = 1;
      u_pieces = ph.g.wk != 0;
      layer_gu[l] = (int)P.size();
      push(ph, "gate_up");
    }
    {
      Phase ph = gemm(u, F, nullptr, false, L.down_w, w, F, PE_RESID);
      ph.g.a_t32 = 1;
      ph.g.a_coh = u_pieces ? 1 : 0;
      resid(ph, mod + 5 * w, nullptr, NS_ROW, next_scale);
      push(ph, "down");
    }
  }
  if (act_off > act_bytes) return fail(RAVEL_E_STATE, "persistent: activation arena too small");
  // final adaptive norm (chunks scale, shift) and output head
  {
    Phase ph = gemm(cur_p, w, shift_of(2 * c.layers), true, m->out_w, D, w, PE_F32);
    ph.g.out_f = b->v;
    ph.g.ldof = D;
    ph.g.bias = m->out_b;
    push(ph, "out_head");
  }
  for (auto& ph : P)
    if (ph.type == PH_GEMM && ph.g.kw == 0) return fail(RAVEL_E_STATE, "persistent: K range too long");
  // Modulation of layer l + 1 (or of the final norm) as side work of layer l's
  // phases before gate/up, in 32-column whole-K items over the conditioning rows, on
  // the blocks those phases leave idle (one item per idle block and phase); the
  // launch before the kernel then computes layer 0's chunk only.  Off when some
  // layer's phases lack the idle blocks, or the shapes do not fit the item.
  {
    if (const char* ev = getenv("RAVEL_NO_FUSED_PROLOGUE")) b->fused_prologue = atoi(ev) == 0;
    bool ok = getenv("RAVEL_NO_SIDE_MOD") == nullptr || atoi(getenv("RAVEL_NO_SIDE_MOD")) == 0;
    ok = ok && w % 128 == 0 && w <= 1024;
    std::vector<PSide> sides(P.size());
    for (auto& sd : sides) memset(&sd, 0, sizeof sd);
    for (int l = 0; l < c.layers && ok; ++l) {
      const bool last = l + 1 == c.layers;
      const size_t col0 = (size_t)(l + 1) * 6 * w;  // the final norm's chunk follows the last layer's
      const int N = last ? 2 * w : 6 * w;
      int remaining = N / 32, next = 0;
      for (int p = layer_first[l]; p < layer_gu[l] && remaining > 0; ++p) {
        const int cap = std::max(0, b->pblocks - P[p].items);
        const int take = std::min(cap, remaining);
        if (take <= 0) continue;
        PSide& sd = sides[p];
        sd.A = (const bf16_t*)b->cond;
        sd.lda = w;
        sd.W = (const bf16_t*)((const char*)m->mod_all_w + col0 * w * 2);
        sd.ldw = w;
        sd.bias = m->mod_all_b + col0;
        sd.out = b->mod + col0;
        sd.ldo = b->mod_ld;
        sd.shift_out[0] = (bf16_t*)shift_of(last ? 2 * c.layers : 2 * (l + 1));
        sd.shift_col[0] = w;
        sd.shift_out[1] = last ? nullptr : (bf16_t*)shift_of(2 * (l + 1) + 1);
        sd.shift_col[1] = 4 * w;
        sd.shift_w = w;
        sd.M = BH;
        sd.N = N;
        sd.K = w;
        sd.item0 = next;
        sd.nitems = take;
        next += take;
        remaining -= take;
      }
      ok = remaining == 0;
    }
    b->side_mod = ok;
    if (ok)
      for (size_t p = 0; p < P.size(); ++p) P[p].side = sides[p];
  }
  // workspaces, patched into the list
  float *gpart, *ao, *aml;
  unsigned* cnt;
  const int Hp = ((H + 15) / 16) * 16;
  RV_TRY(palloc(b, &gpart, part * 4, false));
  RV_TRY(palloc(b, &ao, (size_t)max_attn_parts * Hp * hd * 2, false));  // fp16 split outputs
  RV_TRY(palloc(b, &aml, (size_t)max_attn_parts * Hp * 2 * 4, false));
  // split counters: a range per phase (its tiles, or its (env, head) pairs), each
  // counter used once per launch
  size_t ncnt = 0;
  for (const auto& ph : P) {
    if (ph.type == PH_GEMM && ph.g.ksplit > 1) ncnt += (size_t)tiles(ph.g.N);
    if (ph.type == PH_ATTN && ph.at.nsplit > 1) ncnt += (size_t)B * c.n_q_heads;
  }
  ncnt = std::max(ncnt, (size_t)1);
  b->pgcnt_bytes = ncnt * 4 * kCounterStride;
  b->pcnt_n = (int)ncnt;
  RV_TRY(palloc(b, &cnt, b->pgcnt_bytes, true));
  b->pgcnt = cnt;
  if (!b->hflag) {
    void* h = nullptr;
    HIP_TRY(hipHostMalloc(&h, 64, hipHostMallocMapped));
    b->hflag = (int*)h;
    *b->hflag = 0;
    void* d = nullptr;
    HIP_TRY(hipHostGetDevicePointer(&d, h, 0));
    b->hflag_dev = (int*)d;
  }
  size_t cbase = 0;
  for (auto& ph : P) {
    if (ph.type == PH_GEMM) {
      ph.g.partial = gpart;
      ph.g.counters = cnt + cbase * kCounterStride;
      if (ph.g.ksplit > 1) cbase += (size_t)tiles(ph.g.N);
    } else if (ph.type == PH_ATTN) {
      ph.at.part_o = ao;
      ph.at.part_ml = aml;
      ph.at.counters = cnt + cbase * kCounterStride;
      if (ph.at.nsplit > 1) cbase += (size_t)B * c.n_q_heads;
    }
  }
  RV_TRY(palloc(b, &b->d_phases, P.size() * sizeof(Phase), false));
  HIP_TRY(hipMemcpy(b->d_phases, P.data(), P.size() * sizeof(Phase), hipMemcpyHostToDevice));
  // algorithmic work of the persistent kernel and of each phase (for profiling):
  // weights (bf16) for GEMMs, keys and values (bf16) for attention
  double by = 0, fl = 0;
  b->ph_bytes.assign(P.size(), 0.0);
  b->ph_flops.assign(P.size(), 0.0);
  for (size_t i = 0; i < P.size(); ++i) {
    const Phase& ph = P[i];
    if (ph.type == PH_GEMM) {
      b->ph_bytes[i] = (double)ph.g.N * ph.g.K * 2;
      b->ph_flops[i] = 2.0 * ph.g.M * ph.g.N * ph.g.K;
      if (ph.g.a_mode == PA_XATTN) {  // plus the cross-attention it computes: FOP keys and values
        b->ph_bytes[i] += (double)B * ph.g.x_nf * kvd * 4;
        b->ph_flops[i] += 4.0 * B * c.n_q_heads * H * ph.g.x_nf * hd;
      }
    } else if (ph.type == PH_ATTN) {
      const int nk = ph.at.P + ph.at.S;
      b->ph_bytes[i] = (double)B * nk * kvd * 4;
      b->ph_flops[i] = 4.0 * B * c.n_q_heads * H * nk * hd;
    } else if (ph.type == PH_ROPE) {  // the angle table (the rows stay in L2)
      b->ph_bytes[i] = (double)H * hd * 4;
    }
    if (ph.side.nitems > 0) {  // side work: the modulation weights of its items
      b->ph_bytes[i] += (double)ph.side.nitems * 32 * ph.side.K * 2;
      b->ph_flops[i] += 2.0 * ph.side.M * ph.side.nitems * 32 * ph.side.K;
    }
    by += b->ph_bytes[i];
    fl += b->ph_flops[i];
  }
  b->p_bytes = by;
  b->p_flops = fl;
  RV_TRY(palloc(b, &b->ptimes, (P.size() + 1) * sizeof(unsigned long long), true));
  return RAVEL_OK;
}

ravel_status enqueue_persistent_pass(ravel_buffer* b, const void* fop, hipStream_t s, KernelRecorder* rec,
                                     const PassIn& pin) {
  ravel_model* m = b->m;
  const ravel_config& c = m->cfg;
  const int B = b->B, H = c.horizon, w = c.width, D = c.action_dim, BH = B * H;
  const int kvd = c.n_kv_heads * c.head_dim;
  const double elt = (double)m->elt;
  const bool concat = c.offset_mode == RAVEL_OFFSET_CONCAT;
  const bool adapter = c.offset_mode == RAVEL_OFFSET_ADAPTER;
  const float dbias = pin.lead_bias ? c.delta_bias : 0.f;
  // The rolling step of the MLP offset form in two launches before the layer kernel:
  // (1) the offset conditioning with the input projection (x and its rows' sums of
  // squares), (2) layer 0's modulation, whose epilogue also forms the first norm's p
  // and shift copies, together with the FOP keys / values when they fit the same
  // whole-K kernel.
  const bool prologue2 = b->fused_prologue && b->side_mod && !concat && !adapter && !pin.X && !pin.ages && !pin.ctau && pin.tau_row < 0 &&
                         w % 64 == 0 && plan_gemm(BH, 6 * w, w, false).wholek;
  bool kv_done = false;
  if (prologue2) {
    REC_BEGIN("offset_cond_in_proj", (double)w * w * elt + (double)H * w * 4 + (double)BH * w * elt +
                                         (double)BH * (D + w) * 4 + (double)BH * w * 6,
              2.0 * B * w * w + (double)BH * w * 4 + 2.0 * BH * w * D);
    HIP_TRY(launch_offset_cond_in_proj(b->t, b->t_obs, B, H, dbias, m->d_w1, m->d_b1, (const bf16_t*)m->d_w2, m->d_b2,
                                       w, m->ctau, (bf16_t*)b->cond, b->X, D, m->in_wT, m->in_b, b->x, b->sumsq[0],
                                       s));
    REC_END();
    GemmArgs e = epi_args(EPI_F32);
    e.bias = m->mod_all_b;
    e.out_f = b->mod;
    e.ldo_f = b->mod_ld;
    e.nrm_p = b->pnorm;
    e.nrm_x = b->x;
    e.nrm_shift = b->pshift;
    e.nrm_w = w;
    const bool pair = m->n_ad > 0 && (BH + 15) / 16 == 4 && B * c.n_fop <= 16 &&
                      plan_gemm(B * c.n_fop, m->n_ad * 2 * kvd, w, false).wholek;
    if (pair) {
      e.A = b->cond;
      e.lda = w;
      e.B = m->mod_all_w;
      e.ldb = w;
      e.M = BH;
      e.N = 6 * w;
      e.K = w;
      e.kchunk = w;
      GemmArgs f = epi_args(EPI_T);
      f.out_t = b->kva;
      f.ldo_t = m->n_ad * 2 * kvd;
      f.A = fop;
      f.lda = w;
      f.B = m->kva_w;
      f.ldb = w;
      f.M = B * c.n_fop;
      f.N = m->n_ad * 2 * kvd;
      f.K = w;
      f.kchunk = w;
      REC_BEGIN("mod_layer0_fop_kv",
                ((double)BH * w + 6.0 * w * w + (double)B * c.n_fop * w + (double)f.N * w) * elt +
                    (double)BH * 6 * w * 4 + (double)BH * w * 6 + (double)f.M * f.N * elt,
                2.0 * BH * 6 * w * w + 2.0 * f.M * f.N * w);
      HIP_TRY(launch_gemm_wholek2(e, f, s));
      REC_END();
      kv_done = true;
    } else {
      RV_TRY(run_gemm<bf16_t>(b, s, rec, "mod_layer0", b->cond, w, m->mod_all_w, w, BH, 6 * w, w, e));
    }
  } else if (concat || adapter) {
    REC_BEGIN("offset_value", (double)B * 12, 0.0);
    HIP_TRY(launch_offset_value(pin.X ? nullptr : b->t, b->t_obs, pin.ages, B, H, dbias, b->dval, s));
    REC_END();
    REC_BEGIN("cond_expand", (double)H * w * 4 + (double)BH * w * elt, (double)BH * w * 4);
    HIP_TRY(launch_cond_expand<bf16_t>(nullptr, B, H, w, pin.ctau ? pin.ctau : m->ctau, pin.tau_row, nullptr,
                                       (bf16_t*)b->cond, s));
    REC_END();
  } else {
    // offset MLP and conditioning rows in one launch
    REC_BEGIN("offset_cond", (double)w * w * elt + (double)H * w * 4 + (double)BH * w * elt,
              2.0 * B * w * w + (double)BH * w * 4);
    HIP_TRY(launch_offset_cond(pin.X ? nullptr : b->t, b->t_obs, pin.ages, B, H, dbias, m->d_w1, m->d_b1,
                               (const bf16_t*)m->d_w2, m->d_b2, w, pin.ctau ? pin.ctau : m->ctau, pin.tau_row,
                               (bf16_t*)b->cond, s));
    REC_END();
  }
  if (!prologue2) {
    // every layer's modulation, or layer 0's only when the layer kernel computes the
    // others in blocks its phases leave idle
    GemmArgs e = epi_args(EPI_F32);
    e.bias = m->mod_all_b;
    e.out_f = b->mod;
    e.ldo_f = b->mod_ld;
    RV_TRY(run_gemm<bf16_t>(b, s, rec, b->side_mod ? "mod_layer0" : "mod_all", b->cond, w, m->mod_all_w, w, BH,
                            b->side_mod ? 6 * w : b->mod_ld, w, e));
  }
  if (!prologue2) {
    // input projection with the first layer's norm operands: p of the first norm,
    // the rows' sums of squares, and the bf16 shifts of every norm (chunk 2l and
    // 2l + 1 of layer l, 2L the final norm: 3w apart in the modulation rows,
    // starting at column w)
    InProjNorm nrm;
    nrm.scale = b->mod;
    nrm.ldm = b->mod_ld;
    nrm.p = b->pnorm;
    nrm.sumsq = b->sumsq[0];
    nrm.cvt_in = b->mod + w;
    nrm.cvt_ld = b->mod_ld;
    nrm.cvt_stride = 3 * w;
    nrm.cvt_chunks = b->side_mod ? 2 : 2 * c.layers + 1;
    nrm.cvt_out = b->pshift;
    if (adapter) {
      // the first norm's operands come from the offset form's tokens
      REC_BEGIN("in_proj", (double)BH * (D + w) * 4, 2.0 * BH * w * D);
      HIP_TRY(launch_in_proj(pin.X ? pin.X : b->X, pin.X ? nullptr : b->t, B, H, D, m->in_wT, m->in_b, w, b->x,
                             InProjNorm{}, nullptr, s));
      REC_END();
      RV_TRY(enqueue_offset_adapter<bf16_t>(b, s, rec, pin));
      REC_BEGIN("norm_operands", (double)BH * w * (10 + nrm.cvt_chunks * 6), 0.0);
      HIP_TRY(launch_norm_operands(b->x, BH, w, nrm, s));
      REC_END();
    } else {
      REC_BEGIN("in_proj", (double)BH * (D + w) * 4 + (double)BH * w * (6 + nrm.cvt_chunks * 6),
                2.0 * BH * w * D);
      HIP_TRY(launch_in_proj(pin.X ? pin.X : b->X, pin.X ? nullptr : b->t, B, H, D, m->in_wT, m->in_b, w, b->x,
                             nrm, concat ? b->dval : nullptr, s));
      REC_END();
    }
  }
  if (m->n_ad > 0 && !kv_done) {
    GemmArgs e = epi_args(EPI_T);
    e.out_t = b->kva;
    e.ldo_t = m->n_ad * 2 * kvd;
    RV_TRY(run_gemm<bf16_t>(b, s, rec, "fop_kv", fop, w, m->kva_w, w, B * c.n_fop, m->n_ad * 2 * kvd, w, e));
  }
  REC_BEGIN("persistent_layers", b->p_bytes, b->p_flops);
  HIP_TRY(launch_persistent(b->d_phases, (int)b->phases.size(), b->slot, B, b->pmt, c.head_dim, b->pblocks, b->pbar, b->perr,
                            rec ? b->ptimes : nullptr, b->pgcnt, b->pcnt_n, s));
  REC_END();
  return RAVEL_OK;
}

ravel_status enqueue_persistent_step(ravel_buffer* b, const void* fop, const float* state, float* action,
                                     hipStream_t s, KernelRecorder* rec) {
  const ravel_config& c = b->m->cfg;
  const int B = b->B, H = c.horizon, D = c.action_dim;
  if (state) {
    REC_BEGIN("relative_shift", (double)B * H * D * 8 + (double)B * D * 8, (double)B * H * D * 3);
    HIP_TRY(launch_relative_shift(b->X, b->t, B, H, D, b->rel_mask, state, b->s_prev, b->has_prev, s));
    REC_END();
  }
  RV_TRY(enqueue_persistent_pass(b, fop, s, rec, PassIn{}));
  REC_BEGIN("euler_release", (double)B * H * D * 12 + (double)B * D * 4, (double)B * H * D * 2);
  HIP_TRY(launch_euler_release(b->X, b->v, b->t, B, H, D, b->seed, action, b->ticket, state, b->rel_mask, b->perr,
                               b->hflag_dev, s));
  REC_END();
  return RAVEL_OK;
}

}  // namespace

// c_tau(tau_i) = W_t2 silu(W_t1 emb(tau_i) + b_t1) + b_t2 for tau_i = (i+1)/S, i < S:
// out [S, w] fp32 (synchronous; temporary device memory is freed before it returns).
// With S = H this is the rolling buffer's table; with S Euler steps of a full-horizon
// chunk, step s has tau = (S - s)/S, row S - 1 - s.
static ravel_status flow_time_table(ravel_model* m, int S, float* out) {
  const int w = m->cfg.width;
  const size_t E = m->elt;
  void *emb = nullptr, *hid = nullptr;
  ravel_buffer tmp;  // GEMM workspace only
  tmp.m = m;
  tmp.B = 1;
  const GemmPlan p1 = plan_gemm(S, w, w, false);
  tmp.gpart_elems = p1.part_elems;
  tmp.gcnt_n = std::max(p1.tiles, 1);
  Arena ta;
  void* tarena = nullptr;
  ta.want(&emb, (size_t)S * w * E);
  ta.want(&hid, (size_t)S * w * E);
  ta.want((void**)&tmp.gpart, std::max<size_t>(p1.part_elems, 1) * 4);
  ta.want((void**)&tmp.gcnt, (size_t)tmp.gcnt_n * 4 * kCounterStride);
  ravel_status st = ta.commit(&tarena);
  if (st != RAVEL_OK) return st;
  auto done = [&](ravel_status s2) {
    (void)hipFree(tarena);
    return s2;
  };
  if (hipMemset(tmp.gcnt, 0, (size_t)tmp.gcnt_n * 4 * kCounterStride) != hipSuccess)
    return done(fail(RAVEL_E_HIP, "flow-time table workspace"));
  hipError_t he = m->bf16 ? launch_time_embedding<bf16_t>(S, w, (bf16_t*)emb, 0)
                          : launch_time_embedding<float>(S, w, (float*)emb, 0);
  if (he != hipSuccess) return done(fail(RAVEL_E_HIP, hipGetErrorString(he)));
  GemmArgs e1 = epi_args(EPI_SILU_T);
  e1.bias = m->t_b1;
  e1.out_t = hid;
  e1.ldo_t = w;
  GemmArgs e2 = epi_args(EPI_F32);
  e2.bias = m->t_b2;
  e2.out_f = out;
  e2.ldo_f = w;
  if (m->bf16) {
    st = run_gemm<bf16_t>(&tmp, 0, nullptr, "time1", emb, w, m->t_w1, w, S, w, w, e1);
    if (st == RAVEL_OK) st = run_gemm<bf16_t>(&tmp, 0, nullptr, "time2", hid, w, m->t_w2, w, S, w, w, e2);
  } else {
    st = run_gemm<float>(&tmp, 0, nullptr, "time1", emb, w, m->t_w1, w, S, w, w, e1);
    if (st == RAVEL_OK) st = run_gemm<float>(&tmp, 0, nullptr, "time2", hid, w, m->t_w2, w, S, w, w, e2);
  }
  const hipError_t se = hipDeviceSynchronize();
  if (st != RAVEL_OK) return done(st);
  if (se != hipSuccess) return done(fail(RAVEL_E_HIP, hipGetErrorString(se)));
  return done(RAVEL_OK);
}

// ---------------------------------------------------------------------------
// Fixed device scratch of the allocation-free FOP encoder entry point
// ---------------------------------------------------------------------------
// Staging rows, split-K partials and tickets of ravel_fop_encode_noalloc live in
// this array; every GPU the library runs on holds its own copy until the process
// ends.  Host code never passes the array's name to a kernel: it takes the
// device address from hipGetSymbolAddress, once per device, at model creation.
constexpr size_t kNoAllocScratchBytes = (size_t)16 << 20;
static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

namespace {
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// The current device's address of `scratch` (looked up and cleared on first use).
ravel_status scratch_init_current_device() {
  int dev = 0;
  HIP_TRY(hipGetDevice(&dev));
  if (dev < 0 || dev >= kMaxDevices) return fail(RAVEL_E_STATE, "device index beyond the scratch table");
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (g_scratch_ptr[dev]) return RAVEL_OK;
  void* ptr = nullptr;
  const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
  if (e != hipSuccess || !ptr)
    return fail(RAVEL_E_HIP, std::string("hipGetSymbolAddress(scratch): ") + hipGetErrorString(e));
  HIP_TRY(hipMemset(ptr, 0, kNoAllocScratchBytes));
  HIP_TRY(hipDeviceSynchronize());
  g_scratch_ptr[dev] = ptr;
  return RAVEL_OK;
}

// The FOP stand-in encoder over a batch (shared by both entry points): obs [B, d]
// fp32 -> bf16 staging (bf16 models), hidden = gelu_tanh(W1 obs + b1), tokens =
// W2 hidden + b2; b provides the model, the batch size, the staging rows and the
// GEMM workspace.
ravel_status fop_encode_impl(ravel_buffer* b, const float* obs, void* fop_tokens, hipStream_t s) {
  ravel_model* m = b->m;
  const ravel_config& c = m->cfg;
  const int B = b->B, w = c.width, d = c.fop_obs_dim;
  GemmArgs e1 = epi_args(EPI_GELU_T);
  e1.bias = m->f_b1;
  e1.out_t = b->fhid;
  e1.ldo_t = w;
  GemmArgs e2 = epi_args(EPI_T);
  e2.bias = m->f_b2;
  e2.out_t = fop_tokens;
  e2.ldo_t = c.n_fop * w;
  if (m->bf16) {
    HIP_TRY(launch_convert<bf16_t>(obs, (bf16_t*)b->obs_t, (long long)B * d, s));
    RV_TRY(run_gemm<bf16_t>(b, s, nullptr, "fop1", b->obs_t, d, m->f_w1, d, B, w, d, e1));
    RV_TRY(run_gemm<bf16_t>(b, s, nullptr, "fop2", b->fhid, w, m->f_w2, w, B, c.n_fop * w, w, e2));
  } else {
    RV_TRY(run_gemm<float>(b, s, nullptr, "fop1", obs, d, m->f_w1, d, B, w, d, e1));
    RV_TRY(run_gemm<float>(b, s, nullptr, "fop2", b->fhid, w, m->f_w2, w, B, c.n_fop * w, w, e2));
  }
  return RAVEL_OK;
}
}  // namespace

// ---------------------------------------------------------------------------
// C ABI
// ---------------------------------------------------------------------------
extern "C" {

const char* ravel_last_error(void) { return g_err.c_str(); }

int64_t ravel_model_weight_bytes(const ravel_model* m) { return m ? m->weight_bytes : 0; }

ravel_status ravel_create(const ravel_config* cfgp, const ravel_tensor* weights, int32_t n_weights,
                          ravel_model** out) {
  if (!cfgp || !out || (n_weights > 0 && !weights)) return fail(RAVEL_E_INVALID, "null argument");
  *out = nullptr;
  const ravel_config c = *cfgp;
  if (c.dtype != RAVEL_F32 && c.dtype != RAVEL_BF16) return fail(RAVEL_E_INVALID, "dtype");
  if (c.horizon < 1 || c.horizon > 128) return fail(RAVEL_E_SHAPE, "horizon must be in 1..128");
  if (c.action_dim < 1) return fail(RAVEL_E_SHAPE, "action_dim must be >= 1");
  TensorMap tm;
  for (int i = 0; i < n_weights; ++i) {
    if (!weights[i].name) return fail(RAVEL_E_INVALID, "weight without a name");
    tm.m[weights[i].name] = &weights[i];
  }
  ravel_model* m = new ravel_model();
  m->cfg = c;
  m->bf16 = c.dtype == RAVEL_BF16;
  m->elt = m->bf16 ? 2 : 4;
  (void)hipGetDevice(&m->device);
  auto bail = [&](ravel_status s) {
    if (m->arena) (void)hipFree(m->arena);
    delete m;
    return s;
  };
  const int w = c.width, D = c.action_dim, H = c.horizon;
  if (c.model_kind == RAVEL_ANALYTIC_OT || c.model_kind == RAVEL_ANALYTIC_LINEAR) {
    const char* nm = c.model_kind == RAVEL_ANALYTIC_OT ? "analytic.target" : "analytic.lambda";
    const int64_t n = c.model_kind == RAVEL_ANALYTIC_OT ? D : 1;
    const ravel_tensor* t = tm.get(nm);
    ravel_status st = check_shape(t, nm, {n});
    if (st != RAVEL_OK) return bail(st);
    if (t->dtype != RAVEL_F32) return bail(fail(RAVEL_E_INVALID, "analytic parameter must be fp32"));
    Arena ar;
    ar.want((void**)&m->analytic, n * 4);
    if ((st = ar.commit(&m->arena)) != RAVEL_OK) return bail(st);
    if (hipMemcpy(m->analytic, t->data, n * 4, hipMemcpyDefault) != hipSuccess)
      return bail(fail(RAVEL_E_HIP, "upload analytic parameter"));
    m->weight_bytes = n * 4;
    {
      const ravel_status si = scratch_init_current_device();
      if (si != RAVEL_OK) return bail(si);
    }
    *out = m;
    return RAVEL_OK;
  }
  if (c.model_kind != RAVEL_TRANSFORMER) return bail(fail(RAVEL_E_INVALID, "model_kind"));
  if (c.offset_mode != RAVEL_OFFSET_MLP && c.offset_mode != RAVEL_OFFSET_CONCAT &&
      c.offset_mode != RAVEL_OFFSET_ADAPTER)
    return bail(fail(RAVEL_E_INVALID, "offset_mode"));
  const bool concat = c.offset_mode == RAVEL_OFFSET_CONCAT;
  const bool oadapter = c.offset_mode == RAVEL_OFFSET_ADAPTER;
  if (oadapter && w % 32)
    return bail(fail(RAVEL_E_SHAPE, "RAVEL_OFFSET_ADAPTER needs a width that is a multiple of 32"));
  const int Din = D + (concat ? 1 : 0);  // input features of the action encoder
  const int nq = c.n_q_heads, nkv = c.n_kv_heads, hd = c.head_dim, F = c.mlp_dim, L = c.layers;
  if (w <= 0 || w % 8 || nq <= 0 || nkv <= 0 || nq % nkv || hd % 32 || hd > 256 || F <= 0 || F % 16 ||
      L <= 0 || c.prefix_len < 0 || c.n_fop < 0)
    return bail(fail(RAVEL_E_SHAPE, "invalid transformer config (w%8, hd%32<=256, F%16, nq%nkv)"));
  if (m->bf16 && (H + 15) / 16 > 8) return bail(fail(RAVEL_E_SHAPE, "bf16 attention supports H <= 128"));
  const int qd = nq * hd, kvd = nkv * hd, qkvd = qd + 2 * kvd;
  const int stride = c.fop_stride;
  std::vector<int> ad_of(L, -1);
  int n_ad = 0;
  if (c.n_fop > 0 && stride > 0)
    for (int l = 0; l < L; ++l)
      if (l % stride == stride - 1) ad_of[l] = n_ad++;
  m->n_ad = n_ad;
  m->layers.resize(L);

  // shape checks
  ravel_status st;
#define CHK(name, ...)                                             \
  do {                                                             \
    if ((st = check_shape(tm.get(name), name, {__VA_ARGS__})) != RAVEL_OK) return bail(st); \
  } while (0)
  CHK("in.w", w, Din);
  CHK("in.b", w);
  CHK("time.w1", w, w);
  CHK("time.b1", w);
  CHK("time.w2", w, w);
  CHK("time.b2", w);
  if (c.offset_mode == RAVEL_OFFSET_MLP) {
    CHK("delta.w1", w, 1);
    CHK("delta.b1", w);
    CHK("delta.w2", w, w);
    CHK("delta.b2", w);
  }
  if (oadapter) {
    CHK("at.w1", w, 2 * w + 1);
    CHK("at.b1", w);
    CHK("at.w2", w, w);
    CHK("at.b2", w);
    CHK("ta.w1", w / 4, 2 * w);
    CHK("ta.b1", w / 4);
    CHK("ta.w2", w, w / 4);
    CHK("ta.alpha", 1);
  }
  CHK("final.mod.w", 3 * w, w);
  CHK("final.mod.b", 3 * w);
  CHK("out.w", D, w);
  CHK("out.b", D);
  for (int l = 0; l < L; ++l) {
    const std::string p = "layers." + std::to_string(l) + ".";
    CHK((p + "mod.w").c_str(), 6 * w, w);
    CHK((p + "mod.b").c_str(), 6 * w);
    CHK((p + "qkv.w").c_str(), qkvd, w);
    CHK((p + "o.w").c_str(), w, qd);
    CHK((p + "gate.w").c_str(), F, w);
    CHK((p + "up.w").c_str(), F, w);
    CHK((p + "down.w").c_str(), w, F);
    if (ad_of[l] >= 0) {
      CHK((p + "fop.gamma").c_str(), w);
      CHK((p + "fop.q.w").c_str(), qd, w);
      CHK((p + "fop.kv.w").c_str(), 2 * kvd, w);
      CHK((p + "fop.o.w").c_str(), w, qd);
      CHK((p + "fop.alpha").c_str(), 1);
    }
  }
  m->has_fop_encoder = c.n_fop > 0 && tm.get("fop.w1") != nullptr;
  if (m->has_fop_encoder) {
    CHK("fop.w1", w, c.fop_obs_dim);
    CHK("fop.b1", w);
    CHK("fop.w2", (int64_t)c.n_fop * w, w);
    CHK("fop.b2", (int64_t)c.n_fop * w);
  }
#undef CHK

  // device layout
  const size_t E = m->elt;
  Arena ar;
  ar.want((void**)&m->in_w, (size_t)w * Din * 4);
  ar.want((void**)&m->in_wT, (size_t)w * Din * 4);
  ar.want((void**)&m->in_b, (size_t)w * 4);
  ar.want((void**)&m->ctau, (size_t)H * w * 4);
  ar.want(&m->t_w1, (size_t)w * w * E);
  ar.want(&m->t_w2, (size_t)w * w * E);
  ar.want((void**)&m->t_b1, (size_t)w * 4);
  ar.want((void**)&m->t_b2, (size_t)w * 4);
  ar.want((void**)&m->d_w1, (size_t)w * 4);
  ar.want((void**)&m->d_b1, (size_t)w * 4);
  ar.want((void**)&m->d_w2, (size_t)w * w * E);
  ar.want((void**)&m->d_b2, (size_t)w * 4);
  ar.want(&m->mod_all_w, (size_t)(6 * L + 2) * w * w * E);
  ar.want((void**)&m->mod_all_b, (size_t)(6 * L + 2) * w * 4);
  for (int l = 0; l < L; ++l) {
    LayerW& Lw = m->layers[l];
    ar.want(&Lw.qkv_w, (size_t)qkvd * w * E);
    ar.want(&Lw.o_w, (size_t)w * qd * E);
    ar.want(&Lw.gu_w, (size_t)2 * F * w * E);
    ar.want(&Lw.down_w, (size_t)w * F * E);
    Lw.adapter = ad_of[l];
    if (ad_of[l] >= 0) {
      ar.want((void**)&Lw.gamma, (size_t)w * 4);
      ar.want(&Lw.qa_w, (size_t)qd * w * E);
      ar.want(&Lw.oa_w, (size_t)w * qd * E);
      ar.want((void**)&Lw.alpha, 4);
    }
  }
  if (n_ad > 0) ar.want(&m->kva_w, (size_t)n_ad * 2 * kvd * w * E);
  if (c.rope_base < 0.f || c.rope_base != c.rope_base) return bail(fail(RAVEL_E_INVALID, "rope_base must be >= 0"));
  if (c.rope_base > 0.f) ar.want((void**)&m->rope_cs, (size_t)H * hd * 4);
  if (oadapter) {
    m->at_kz = 2 * w + 64;
    ar.want(&m->at_w1, (size_t)w * m->at_kz * E);
    ar.want(&m->at_w2, (size_t)w * w * E);
    ar.want(&m->ta_w1, (size_t)(w / 4) * 2 * w * E);
    ar.want(&m->ta_w2, (size_t)w * (w / 4) * E);
    ar.want((void**)&m->at_b1, (size_t)w * 4);
    ar.want((void**)&m->at_b2, (size_t)w * 4);
    ar.want((void**)&m->ta_b1, (size_t)(w / 4) * 4);
    ar.want((void**)&m->ta_alpha, 4);
  }
  ar.want(&m->out_w, (size_t)D * w * E);
  ar.want((void**)&m->out_b, (size_t)D * 4);
  if (m->has_fop_encoder) {
    ar.want(&m->f_w1, (size_t)w * c.fop_obs_dim * E);
    ar.want((void**)&m->f_b1, (size_t)w * 4);
    ar.want(&m->f_w2, (size_t)c.n_fop * w * w * E);
    ar.want((void**)&m->f_b2, (size_t)c.n_fop * w * 4);
  }
  m->arena_bytes = ar.off;
  if ((st = ar.commit(&m->arena)) != RAVEL_OK) return bail(st);
  for (int l = 0; l < L; ++l) {
    m->layers[l].mod_w = (char*)m->mod_all_w + (size_t)l * 6 * w * w * E;
    m->layers[l].mod_b = m->mod_all_b + (size_t)l * 6 * w;
  }
  m->fmod_w = (char*)m->mod_all_w + (size_t)L * 6 * w * w * E;
  m->fmod_b = m->mod_all_b + (size_t)L * 6 * w;

  // staging (fp32 + converted bf16) for uploads
  Staging stg;
  stg.S = (size_t)std::max<int64_t>((int64_t)6 * w * w, (int64_t)c.n_fop * w * w);
  stg.S = std::min<size_t>(stg.S, (size_t)64 << 20);
  stg.S = std::max<size_t>(stg.S, (size_t)2 * F * w);
  void* staging = nullptr;
  if (hipMalloc(&staging, stg.S * 6 + 512) != hipSuccess) return bail(fail(RAVEL_E_NOMEM, "staging"));
  stg.f = (float*)staging;
  stg.h = (bf16_t*)((char*)staging + align_up(stg.S * 4, 256));
  auto up = [&](const char* name, void* dst, bool model_dtype) {
    return upload_all(tm.get(name), model_dtype && m->bf16, dst, stg);
  };
  auto done = [&](ravel_status s2) {
    (void)hipFree(staging);
    return s2;
  };
#define UP(name, dst, md)                                     \
  do {                                                        \
    if ((st = up(name, dst, md)) != RAVEL_OK) return bail(done(st)); \
  } while (0)
  UP("in.w", m->in_w, false);
  if (launch_transpose_f32(m->in_w, w, Din, m->in_wT, 0) != hipSuccess)
    return bail(done(fail(RAVEL_E_HIP, "in.w transpose")));
  UP("in.b", m->in_b, false);
  if (m->rope_cs) {
    // rotary table: slot i at position P + i, pair d at base^(-2d/hd), in float64
    std::vector<float> cs((size_t)H * hd);
    for (int i = 0; i < H; ++i)
      for (int d = 0; d < hd / 2; ++d) {
        const double ang = (double)(c.prefix_len + i) * pow((double)c.rope_base, -2.0 * d / hd);
        cs[((size_t)i * (hd / 2) + d) * 2] = (float)cos(ang);
        cs[((size_t)i * (hd / 2) + d) * 2 + 1] = (float)sin(ang);
      }
    if (hipMemcpy(m->rope_cs, cs.data(), cs.size() * 4, hipMemcpyHostToDevice) != hipSuccess)
      return bail(done(fail(RAVEL_E_HIP, "rope table")));
  }
  if (oadapter) {
    // action-time MLP, first layer: [w, 2w + 1] rows placed in [w, at_kz] with zero padding
    const size_t src_row = (size_t)(2 * w + 1) * E, dst_row = (size_t)m->at_kz * E;
    void* tmp = nullptr;
    if (hipMalloc(&tmp, (size_t)w * src_row) != hipSuccess) return bail(done(fail(RAVEL_E_NOMEM, "at.w1 staging")));
    st = up("at.w1", tmp, true);
    if (st == RAVEL_OK && (hipMemset(m->at_w1, 0, (size_t)w * dst_row) != hipSuccess ||
                           hipMemcpy2D(m->at_w1, dst_row, tmp, src_row, src_row, w, hipMemcpyDeviceToDevice) !=
                               hipSuccess))
      st = fail(RAVEL_E_HIP, "at.w1 upload");
    (void)hipFree(tmp);
    if (st != RAVEL_OK) return bail(done(st));
    UP("at.b1", m->at_b1, false);
    UP("at.w2", m->at_w2, true);
    UP("at.b2", m->at_b2, false);
    UP("ta.w1", m->ta_w1, true);
    UP("ta.b1", m->ta_b1, false);
    UP("ta.w2", m->ta_w2, true);
    UP("ta.alpha", m->ta_alpha, false);
  }
  if (c.offset_mode == RAVEL_OFFSET_MLP) {
    UP("delta.w1", m->d_w1, false);
    UP("delta.b1", m->d_b1, false);
    UP("delta.w2", m->d_w2, true);
    UP("delta.b2", m->d_b2, false);
  }
  for (int l = 0; l < L; ++l) {
    LayerW& Lw = m->layers[l];
    const std::string p = "layers." + std::to_string(l) + ".";
    UP((p + "mod.w").c_str(), Lw.mod_w, true);
    UP((p + "mod.b").c_str(), Lw.mod_b, false);
    UP((p + "qkv.w").c_str(), Lw.qkv_w, true);
    UP((p + "o.w").c_str(), Lw.o_w, true);
    UP((p + "down.w").c_str(), Lw.down_w, true);
    // gate/up interleave: dst row 32b + j <- gate row 16b + j, dst row 32b + 16 + j <- up row 16b + j
    {
      const ravel_tensor* g = tm.get(p + "gate.w");
      const ravel_tensor* u = tm.get(p + "up.w");
      if ((st = upload_rows(g, 0, F, w, m->bf16, Lw.gu_w, [](int64_t r) { return (r / 16) * 32 + (r % 16); },
                            stg)) != RAVEL_OK)
        return bail(done(st));
      if ((st = upload_rows(u, 0, F, w, m->bf16, Lw.gu_w,
                            [](int64_t r) { return (r / 16) * 32 + 16 + (r % 16); }, stg)) != RAVEL_OK)
        return bail(done(st));
    }
    if (Lw.adapter >= 0) {
      UP((p + "fop.gamma").c_str(), Lw.gamma, false);
      UP((p + "fop.q.w").c_str(), Lw.qa_w, true);
      UP((p + "fop.o.w").c_str(), Lw.oa_w, true);
      UP((p + "fop.alpha").c_str(), Lw.alpha, false);
      void* dst = (char*)m->kva_w + (size_t)Lw.adapter * 2 * kvd * w * E;
      UP((p + "fop.kv.w").c_str(), dst, true);
    }
  }
  {
    // final modulation: only the scale and shift chunks (rows 0 .. 2w) are used
    const ravel_tensor* fw = tm.get("final.mod.w");
    if ((st = upload_rows(fw, 0, 2 * w, w, m->bf16, m->fmod_w, [](int64_t r) { return r; }, stg)) !=
        RAVEL_OK)
      return bail(done(st));
    const ravel_tensor* fb = tm.get("final.mod.b");
    if (hipMemcpy(m->fmod_b, fb->data, (size_t)2 * w * 4, hipMemcpyDefault) != hipSuccess)
      return bail(done(fail(RAVEL_E_HIP, "final.mod.b")));
  }
  UP("out.w", m->out_w, true);
  UP("out.b", m->out_b, false);
  if (m->has_fop_encoder) {
    UP("fop.w1", m->f_w1, true);
    UP("fop.b1", m->f_b1, false);
    UP("fop.w2", m->f_w2, true);
    UP("fop.b2", m->f_b2, false);
  }

  // flow-time conditioning c_tau(i) = W_t2 silu(W_t1 emb(tau_i) + b_t1) + b_t2, once per model
  UP("time.w1", m->t_w1, true);
  UP("time.w2", m->t_w2, true);
  UP("time.b1", m->t_b1, false);
  UP("time.b2", m->t_b2, false);
  if ((st = flow_time_table(m, H, m->ctau)) != RAVEL_OK) return bail(done(st));
  (void)hipFree(staging);
#undef UP
  if (hipDeviceSynchronize() != hipSuccess) return bail(fail(RAVEL_E_HIP, "create sync"));
  // algorithmic weight bytes streamed by one step (time MLP excluded: precomputed)
  int64_t wb = (int64_t)w * Din * 4 + (c.offset_mode == RAVEL_OFFSET_MLP ? (int64_t)w * w * E : 0);
  if (oadapter) wb += ((int64_t)w * m->at_kz + (int64_t)w * w + (int64_t)w * w / 2 + (int64_t)w * w / 4) * E;
  for (int l = 0; l < L; ++l) {
    wb += (int64_t)(6 * w + qkvd) * w * E + (int64_t)w * qd * E + (int64_t)3 * F * w * E + 6 * w * 4;
    if (ad_of[l] >= 0) wb += (int64_t)(2 * qd + 2 * kvd) * w * E;
  }
  wb += (int64_t)2 * w * w * E + (int64_t)D * w * E;
  m->weight_bytes = wb;
  {
    const ravel_status si = scratch_init_current_device();
    if (si != RAVEL_OK) return bail(si);
  }
  *out = m;
  return RAVEL_OK;
}

void ravel_destroy(ravel_model* m) {
  if (!m) return;
  if (m->arena) (void)hipFree(m->arena);
  delete m;
}

ravel_status ravel_buffer_create(ravel_model* m, int32_t batch, uint64_t seed, ravel_buffer** out) {
  if (!m || !out) return fail(RAVEL_E_INVALID, "null argument");
  if (batch < 1) return fail(RAVEL_E_SHAPE, "batch must be >= 1");
  *out = nullptr;
  if (const char* ev = getenv("RAVEL_COOPERATIVE"))
    if (atoi(ev) != 0)
      return fail(RAVEL_E_INVALID, "RAVEL_COOPERATIVE: the cooperative launch of the layers' kernel is not supported "
                                   "(an ordinary launch with bounded waits is used)");
  const ravel_config& c = m->cfg;
  ravel_buffer* b = new ravel_buffer();
  b->m = m;
  b->B = batch;
  b->seed = seed;
  const int B = batch, H = c.horizon, D = c.action_dim, BH = B * H;
  const size_t E = m->elt;
  Arena ar;
  ar.want((void**)&b->X, (size_t)BH * D * 4);
  ar.want((void**)&b->t, 8);
  ar.want((void**)&b->t_obs, (size_t)B * 8);
  ar.want((void**)&b->slot, (size_t)B * 4);
  ar.want((void**)&b->ticket, 4);
  ar.want((void**)&b->v, (size_t)BH * D * 4);
  ar.want((void**)&b->trainX, (size_t)BH * D * 4);
  ar.want((void**)&b->rel_mask, (size_t)D * 4);
  ar.want((void**)&b->s_prev, (size_t)B * D * 4);
  ar.want((void**)&b->has_prev, (size_t)B * 4);
  ar.want((void**)&b->dbg_flag, 4);
  size_t part_elems = 0, cnt = 1;
  if (c.model_kind == RAVEL_TRANSFORMER) {
    const int w = c.width, qd = c.n_q_heads * c.head_dim, kvd = c.n_kv_heads * c.head_dim;
    const int qkvd = qd + 2 * kvd, F = c.mlp_dim;
    b->ctx_elems = (size_t)c.layers * c.prefix_len * kvd;
    ar.want(&b->ctx_k, 2 * (size_t)B * b->ctx_elems * E);
    ar.want(&b->ctx_v, 2 * (size_t)B * b->ctx_elems * E);
    ar.want((void**)&b->x, (size_t)BH * w * 4);
    ar.want(&b->cond, (size_t)BH * w * E);
    ar.want(&b->h1, (size_t)B * w * E);
    ar.want((void**)&b->dvec, (size_t)B * w * 4);
    ar.want((void**)&b->dval, (size_t)B * 8);
    if (m->at_kz > 0) {
      ar.want(&b->tz, (size_t)BH * m->at_kz * E);
      ar.want(&b->th, (size_t)BH * w * E);
    }
    // few rows: every layer's modulation comes from one GEMM at the start of the step
    // Few rows, or rows grouped by offset conditioning: every layer's modulation
    // comes from one GEMM at the start of the step (on the groups' rows only).
    b->cgroups = BH > 64 && B > 1 && B <= kCondGroupsMaxB;
    b->mod_all = BH <= 64 || b->cgroups;
    b->mod_ld = b->mod_all ? (6 * c.layers + 2) * w : 6 * w;
    if (b->cgroups) {
      ar.want((void**)&b->cgrp, (size_t)B * 4);
      ar.want((void**)&b->crowmap, (size_t)BH * 4);
      ar.want((void**)&b->crows, 16);
    }
    ar.want((void**)&b->mod, (size_t)BH * b->mod_ld * 4);
    ar.want(&b->y, (size_t)BH * w * E);
    ar.want(&b->qkv, (size_t)BH * qkvd * E);
    ar.want(&b->att, (size_t)BH * qd * E);
    ar.want(&b->qa, (size_t)BH * qd * E);
    if (m->n_ad > 0) ar.want(&b->kva, (size_t)B * c.n_fop * m->n_ad * 2 * kvd * E);
    ar.want(&b->u, (size_t)BH * F * E);
    ar.want((void**)&b->fmod, (size_t)BH * 2 * w * 4);
    ar.want(&b->fhid, (size_t)B * w * E);
    ar.want(&b->obs_t, (size_t)B * std::max(c.fop_obs_dim, 1) * E);
    // GEMM split-K workspace: the largest plan of the step
    struct Shape { int M, N, K; bool geglu; };
    std::vector<Shape> shapes = {{B, w, w, false}, {BH, 6 * w, w, false}, {BH, (6 * c.layers + 2) * w, w, false},
                                 {BH, qkvd, w, false},
                                 {BH, w, qd, false}, {BH, qd, w, false}, {BH, 2 * F, w, true},
                                 {BH, w, F, false}, {BH, 2 * w, w, false}, {BH, D, w, false},
                                 {B, w, std::max(c.fop_obs_dim, 8), false}, {B, c.n_fop * w, w, false}};
    if (m->n_ad > 0) shapes.push_back({B * c.n_fop, m->n_ad * 2 * kvd, w, false});
    if (m->at_kz > 0) {
      shapes.push_back({BH, w, m->at_kz, false});
      shapes.push_back({BH, w / 4, 2 * w, false});
      shapes.push_back({BH, w, w / 4, false});
    }
    for (auto& s : shapes) {
      if (s.N <= 0 || s.M <= 0) continue;
      const GemmPlan p = plan_gemm(s.M, s.N, s.K, s.geglu);
      part_elems = std::max(part_elems, p.part_elems);
      cnt = std::max(cnt, (size_t)p.tiles);
    }
    // attention key split: aim for ~256 blocks when B * nq is small, >= 64 keys per split
    const int nkeys = c.prefix_len + H;
    const int blocks = B * c.n_q_heads;
    int ns = 1;
    if (m->bf16 && blocks < 64) {
      // a few blocks per CU-group at batch 1: split keys, >= 128 keys per split; the
      // merge keeps nsplit x H softmax weights in the 32-key tile's LDS
      ns = std::min((nkeys + 127) / 128, (64 + blocks - 1) / blocks);
      const int cap = 32 * (c.head_dim + 8) / 2 / H;
      ns = std::max(1, std::min(ns, cap));
    }
    int kps = ((nkeys + ns - 1) / ns + 31) / 32 * 32;
    ns = (nkeys + kps - 1) / kps;
    b->attn_nsplit = ns;
    b->attn_kps = kps;
    if (ns > 1) {
      const int Hp = (H + 15) / 16 * 16;
      ar.want((void**)&b->apart_o, (size_t)blocks * ns * Hp * c.head_dim * 4);
      ar.want((void**)&b->apart_ml, (size_t)blocks * ns * Hp * 2 * 4);
    }
    ar.want((void**)&b->acnt, (size_t)blocks * 4 * kCounterStride);
  }
  ar.want((void**)&b->gpart, std::max<size_t>(part_elems, 1) * 4);
  ar.want((void**)&b->gcnt, cnt * 4 * kCounterStride);
  b->gpart_elems = part_elems;
  b->gcnt_n = (int)cnt;
  ravel_status st = ar.commit(&b->arena);
  if (st != RAVEL_OK) {
    delete b;
    return st;
  }
  auto bail = [&](ravel_status s2) {
    (void)hipFree(b->arena);
    delete b;
    return s2;
  };
  if (hipMemset(b->arena, 0, ar.off) != hipSuccess) return bail(fail(RAVEL_E_HIP, "memset"));
  if (launch_ring_init(b->X, B, H, D, seed, 0) != hipSuccess) return bail(fail(RAVEL_E_HIP, "ring init"));
  if (hipDeviceSynchronize() != hipSuccess) return bail(fail(RAVEL_E_HIP, "buffer create sync"));
  b->active.assign(B, 0);
  b->has_ctx.assign(B, 0);
  b->tobs_host.assign(B, 0);
  b->pending.resize(B);
  b->retire.resize(B);
  b->retire_valid.assign(B, 0);
  for (int e = 0; e < B; ++e) {
    if (hipEventCreateWithFlags(&b->pending[e].ready, hipEventDisableTiming) != hipSuccess ||
        hipEventCreateWithFlags(&b->retire[e], hipEventDisableTiming) != hipSuccess)
      return bail(fail(RAVEL_E_HIP, "event create"));
  }
  if (hipStreamCreateWithFlags(&b->cap_stream, hipStreamNonBlocking) != hipSuccess)
    return bail(fail(RAVEL_E_HIP, "stream create"));
  if (persistent_eligible(b)) {
    if (build_persistent(b) == RAVEL_OK) {
      b->persistent = true;
    } else {
      for (void* p : b->pallocs) (void)hipFree(p);
      b->pallocs.clear();
      b->d_phases = nullptr;
      b->pbar = nullptr;
      b->perr = nullptr;
      b->persistent = false;
    }
    if (const char* ev = getenv("RAVEL_NO_PERSISTENT")) b->persistent = b->persistent && atoi(ev) == 0;
  }
  if (const char* ev = getenv("RAVEL_SYNC_CONTEXT")) b->sync_ctx = atoi(ev) != 0;
  if (const char* ev = getenv("RAVEL_NO_GRAPH")) b->use_graph = atoi(ev) == 0;
  if (const char* ev = getenv("RAVEL_DEBUG")) b->debug = atoi(ev) != 0;
  *out = b;
  return RAVEL_OK;
}

void ravel_buffer_destroy(ravel_buffer* b) {
  if (!b) return;
  (void)hipDeviceSynchronize();
  for (auto& g : b->graphs) {
    (void)hipGraphExecDestroy(g.exec);
    (void)hipGraphDestroy(g.graph);
  }
  for (int e = 0; e < b->B; ++e) {
    if (b->pending[e].ready) (void)hipEventDestroy(b->pending[e].ready);
    if (b->retire[e]) (void)hipEventDestroy(b->retire[e]);
  }
  if (b->cap_stream) (void)hipStreamDestroy(b->cap_stream);
  if (b->hflag) (void)hipHostFree(b->hflag);
  for (void* p : b->pallocs) (void)hipFree(p);
  for (auto& kv : b->full_tables) (void)hipFree(kv.second);
  if (b->arena) (void)hipFree(b->arena);
  delete b;
}

ravel_status ravel_buffer_set_option(ravel_buffer* b, int32_t option, int64_t value) {
  if (!b) return fail(RAVEL_E_INVALID, "null buffer");
  std::lock_guard<std::mutex> lk(b->mu);
  switch (option) {
    case RAVEL_OPT_SYNC_CONTEXT: b->sync_ctx = value != 0; return RAVEL_OK;
    case RAVEL_OPT_USE_GRAPH: b->use_graph = value != 0; return RAVEL_OK;
    case RAVEL_OPT_DEBUG: b->debug = value != 0; return RAVEL_OK;
    case RAVEL_OPT_PERSISTENT:
      if (value != 0 && !b->d_phases) return fail(RAVEL_E_STATE, "persistent path not available for this model/batch");
      b->persistent = value != 0;
      return RAVEL_OK;
    case RAVEL_OPT_FAIL_LAYERS: {
      if (!b->perr) return fail(RAVEL_E_STATE, "no persistent layers' kernel on this buffer");
      HIP_TRY(hipDeviceSynchronize());
      const int word = value != 0 ? 4 : 0;
      HIP_TRY(hipMemcpy(b->perr, &word, 4, hipMemcpyHostToDevice));
      return RAVEL_OK;
    }
    default: return fail(RAVEL_E_INVALID, "unknown option");
  }
}

ravel_status ravel_context_acquire(ravel_buffer* b, int32_t env, void** k, void** v, void* producer) {
  if (!b || !k || !v) return fail(RAVEL_E_INVALID, "null argument");
  if (b->m->cfg.model_kind != RAVEL_TRANSFORMER) return fail(RAVEL_E_STATE, "analytic models have no context");
  if (env < 0 || env >= b->B) return fail(RAVEL_E_INVALID, "env out of range");
  std::lock_guard<std::mutex> lk(b->mu);
  return acquire_locked(b, env, k, v, (hipStream_t)producer);
}

ravel_status ravel_set_context(ravel_buffer* b, int32_t env, const void* k, const void* v, int64_t t_obs,
                               void* producer) {
  if (!b) return fail(RAVEL_E_INVALID, "null buffer");
  if (b->m->cfg.model_kind != RAVEL_TRANSFORMER) return fail(RAVEL_E_STATE, "analytic models have no context");
  if (env < -1 || env >= b->B) return fail(RAVEL_E_INVALID, "env out of range");
  if ((k == nullptr) != (v == nullptr)) return fail(RAVEL_E_INVALID, "k and v must both be given or both NULL");
  if (env == -1 && !k) return fail(RAVEL_E_INVALID, "env = -1 needs k and v ([B, L, P, n_kv, hd])");
  hipStream_t ps = (hipStream_t)producer;
  std::lock_guard<std::mutex> lk(b->mu);
  const int e0 = env < 0 ? 0 : env, e1 = env < 0 ? b->B : env + 1;
  // every env's t_obs is checked before anything is copied: all or none
  for (int e = e0; e < e1; ++e) {
    int64_t latest = b->has_ctx[e] ? b->tobs_host[e] : INT64_MIN;
    if (b->pending[e].valid) latest = std::max(latest, b->pending[e].t_obs);
    if (t_obs < latest) return fail(RAVEL_E_STATE, "t_obs must not decrease per env (env " + std::to_string(e) + ")");
  }
  const size_t bytes = b->ctx_elems * b->m->elt;
  for (int e = e0; e < e1; ++e) {
    if (k) {
      void *dk, *dv;
      RV_TRY(acquire_locked(b, e, &dk, &dv, ps));
      const size_t src = env < 0 ? (size_t)e * bytes : 0;  // [B, L, P, n_kv, hd]: env e's block
      HIP_TRY(hipMemcpyAsync(dk, (const char*)k + src, bytes, hipMemcpyDefault, ps));
      HIP_TRY(hipMemcpyAsync(dv, (const char*)v + src, bytes, hipMemcpyDefault, ps));
    }
    HIP_TRY(hipEventRecord(b->pending[e].ready, ps));
    b->pending[e].valid = true;
    b->pending[e].t_obs = t_obs;
  }
  return RAVEL_OK;
}

namespace {
// After a failed launch of the layers' kernel (device idle): the blocks that gave
// up left the barrier and split counters behind, and every launch since returned
// at once (the error word is sticky): re-arm all of them, clear the word and the
// host flag, and take the step counter back from the device (failed steps did not
// advance it).
ravel_status persistent_rearm(ravel_buffer* b) {
  HIP_TRY(hipMemset(b->pbar, 0, kBarrierWords * 4));
  if (b->pgcnt) HIP_TRY(hipMemset(b->pgcnt, 0, b->pgcnt_bytes));
  HIP_TRY(hipMemset(b->perr, 0, 64));
  HIP_TRY(hipDeviceSynchronize());
  if (b->hflag) __atomic_store_n(b->hflag, 0, __ATOMIC_RELEASE);
  int64_t t = 0;
  HIP_TRY(hipMemcpy(&t, b->t, 8, hipMemcpyDeviceToHost));
  b->t_host = t;
  return RAVEL_OK;
}

ravel_status check_persistent_error(ravel_buffer* b) {
  if (!b->perr) return RAVEL_OK;
  int e = 0;
  HIP_TRY(hipMemcpy(&e, b->perr, 4, hipMemcpyDeviceToHost));
  if (e) {
    RV_TRY(persistent_rearm(b));
    return fail(RAVEL_E_HIP, "persistent kernel: a grid barrier timed out; the steps since released NaN actions "
                             "and left the ring and t unchanged");
  }
  return RAVEL_OK;
}

// Called at the start of every call that enqueues work (caller holds the mutex): a
// release kernel found the layers' kernel failed and raised the pinned host flag
// (no synchronisation unless it is up).
ravel_status check_failed_launch(ravel_buffer* b) {
  if (!b->hflag || __atomic_load_n(b->hflag, __ATOMIC_ACQUIRE) == 0) return RAVEL_OK;
  HIP_TRY(hipDeviceSynchronize());
  RV_TRY(persistent_rearm(b));
  return fail(RAVEL_E_HIP, "persistent kernel: a grid barrier timed out; the steps since released NaN actions "
                           "and left the ring and t unchanged");
}
}  // namespace

ravel_status ravel_full_denoise(ravel_buffer* b, int32_t steps, const void* fop, const float* noise, float* chunk,
                                void* stream) {
  if (!b || !noise || !chunk) return fail(RAVEL_E_INVALID, "null argument");
  ravel_model* m = b->m;
  const ravel_config& c = m->cfg;
  const int B = b->B, H = c.horizon, D = c.action_dim;
  if (steps < 1 || steps > kMaxFullSteps) return fail(RAVEL_E_SHAPE, "steps must be in 1..1024");
  if (c.model_kind == RAVEL_TRANSFORMER && m->n_ad > 0 && !fop)
    return fail(RAVEL_E_INVALID, "fop_tokens required: the model has FOP adapters");
  if (fop && ((uintptr_t)fop % 16)) return fail(RAVEL_E_INVALID, "fop_tokens must be 16-byte aligned");
  hipStream_t s = (hipStream_t)stream;
  std::lock_guard<std::mutex> lk(b->mu);
  RV_TRY(check_failed_launch(b));
  const float* table = nullptr;
  if (c.model_kind == RAVEL_TRANSFORMER) {
    // contexts: the latest available ones, published exactly as a rolling step would
    RV_TRY(apply_publishes(b, s));
    for (int e = 0; e < B; ++e)
      if (!b->has_ctx[e]) return fail(RAVEL_E_STATE, "env " + std::to_string(e) + " has no context yet");
    auto it = b->full_tables.find(steps);
    if (it == b->full_tables.end()) {
      float* t = nullptr;
      HIP_TRY(hipMalloc(&t, (size_t)steps * c.width * 4));
      const ravel_status st = flow_time_table(m, steps, t);
      if (st != RAVEL_OK) {
        (void)hipFree(t);
        return st;
      }
      it = b->full_tables.emplace(steps, t).first;
    }
    table = it->second;
  }
  const size_t bytes = (size_t)B * H * D * 4;
  if (chunk != noise) HIP_TRY(hipMemcpyAsync(chunk, noise, bytes, hipMemcpyDeviceToDevice, s));
  const float dt = 1.0f / (float)steps;
  for (int k = 0; k < steps; ++k) {
    // step k: every slot at tau = (steps - k) / steps, row steps - 1 - k of the table
    if (c.model_kind == RAVEL_TRANSFORMER) {
      PassIn pin;
      pin.X = chunk;
      pin.ctau = table;
      pin.tau_row = steps - 1 - k;
      pin.tau_den = steps;
      if (b->persistent)
        RV_TRY(enqueue_persistent_pass(b, fop, s, nullptr, pin));
      else if (m->bf16)
        RV_TRY(enqueue_transformer<bf16_t>(b, fop, s, nullptr, pin));
      else
        RV_TRY(enqueue_transformer<float>(b, fop, s, nullptr, pin));
    } else {
      HIP_TRY(launch_analytic_velocity(c.model_kind, chunk, nullptr, B, H, D, m->analytic,
                                       (float)(steps - k) / (float)steps, nullptr, nullptr, b->v, s));
    }
    HIP_TRY(launch_euler_chunk(chunk, b->v, B, H, D, dt, s));
  }
  return RAVEL_OK;
}

ravel_status ravel_train_loss(ravel_buffer* b, const float* target, const float* noise, const int64_t* ages,
                              const void* fop, float* loss, float* v_out, void* stream) {
  if (!b || !target || !noise || !ages || !loss) return fail(RAVEL_E_INVALID, "null argument");
  ravel_model* m = b->m;
  const ravel_config& c = m->cfg;
  const int B = b->B, H = c.horizon, D = c.action_dim;
  if (c.model_kind == RAVEL_TRANSFORMER && m->n_ad > 0 && !fop)
    return fail(RAVEL_E_INVALID, "fop_tokens required: the model has FOP adapters");
  if (fop && ((uintptr_t)fop % 16)) return fail(RAVEL_E_INVALID, "fop_tokens must be 16-byte aligned");
  hipStream_t s = (hipStream_t)stream;
  std::lock_guard<std::mutex> lk(b->mu);
  RV_TRY(check_failed_launch(b));
  if (c.model_kind == RAVEL_TRANSFORMER) {
    RV_TRY(apply_publishes(b, s));
    for (int e = 0; e < B; ++e)
      if (!b->has_ctx[e]) return fail(RAVEL_E_STATE, "env " + std::to_string(e) + " has no context yet");
  }
  HIP_TRY(launch_train_buffer(target, noise, B, H, D, b->trainX, s));
  if (c.model_kind == RAVEL_TRANSFORMER) {
    PassIn pin;
    pin.X = b->trainX;
    pin.ages = ages;
    pin.lead_bias = false;
    if (b->persistent)
      RV_TRY(enqueue_persistent_pass(b, fop, s, nullptr, pin));
    else if (m->bf16)
      RV_TRY(enqueue_transformer<bf16_t>(b, fop, s, nullptr, pin));
    else
      RV_TRY(enqueue_transformer<float>(b, fop, s, nullptr, pin));
  } else {
    HIP_TRY(launch_analytic_velocity(c.model_kind, b->trainX, nullptr, B, H, D, m->analytic, 0.f, nullptr, nullptr,
                                     b->v, s));
  }
  HIP_TRY(launch_train_loss(b->v, target, noise, B, H, D, loss, s));
  if (v_out) HIP_TRY(hipMemcpyAsync(v_out, b->v, (size_t)B * H * D * 4, hipMemcpyDeviceToDevice, s));
  return RAVEL_OK;
}

static ravel_status step_impl(ravel_buffer* b, const void* fop, const float* state, float* action, void* stream) {
  if (!b || !action) return fail(RAVEL_E_INVALID, "null argument");
  if (b->relative && !state) return fail(RAVEL_E_STATE, "relative actions: use ravel_step_state with the robot state");
  if (!b->relative && state) return fail(RAVEL_E_STATE, "no relative dimensions set (ravel_set_relative_dims)");
  ravel_model* m = b->m;
  const ravel_config& c = m->cfg;
  if (c.model_kind == RAVEL_TRANSFORMER && m->n_ad > 0 && !fop)
    return fail(RAVEL_E_INVALID, "fop_tokens required: the model has FOP adapters");
  if (fop && ((uintptr_t)fop % 16)) return fail(RAVEL_E_INVALID, "fop_tokens must be 16-byte aligned");
  hipStream_t s = (hipStream_t)stream;
  std::lock_guard<std::mutex> lk(b->mu);
  RV_TRY(check_failed_launch(b));
  if (c.model_kind == RAVEL_TRANSFORMER) {
    RV_TRY(apply_publishes(b, s));
    for (int e = 0; e < b->B; ++e)
      if (!b->has_ctx[e]) return fail(RAVEL_E_STATE, "env " + std::to_string(e) + " has no context yet");
  }
  if (b->use_graph) {
    // one captured graph per (fop, state, action) pointer set and execution path
    GraphEntry* ge = nullptr;
    for (auto& g : b->graphs)
      if (g.fop == fop && g.state == state && g.action == action && g.persistent == b->persistent) ge = &g;
    if (!ge) {
      GraphEntry g{fop, state, action, b->persistent, nullptr, nullptr};
      HIP_TRY(hipStreamBeginCapture(b->cap_stream, hipStreamCaptureModeRelaxed));
      ravel_status st = b->persistent ? enqueue_persistent_step(b, fop, state, action, b->cap_stream, nullptr)
                                      : enqueue_step(b, fop, state, action, b->cap_stream, nullptr);
      hipGraph_t graph = nullptr;
      hipError_t he = hipStreamEndCapture(b->cap_stream, &graph);
      if (st != RAVEL_OK) return st;
      if (he != hipSuccess) return fail(RAVEL_E_HIP, std::string("capture: ") + hipGetErrorString(he));
      g.graph = graph;
      HIP_TRY(hipGraphInstantiate(&g.exec, graph, nullptr, nullptr, 0));
      b->graphs.push_back(g);
      ge = &b->graphs.back();
    }
    HIP_TRY(hipGraphLaunch(ge->exec, s));
  } else if (b->persistent) {
    RV_TRY(enqueue_persistent_step(b, fop, state, action, s, nullptr));
  } else {
    RV_TRY(enqueue_step(b, fop, state, action, s, nullptr));
  }
  b->t_host += 1;
  if (b->debug) {
    HIP_TRY(hipStreamSynchronize(s));
    HIP_TRY(hipMemset(b->dbg_flag, 0, 4));
    HIP_TRY(launch_check_finite(b->X, (long long)b->B * c.horizon * c.action_dim, b->dbg_flag, s));
    HIP_TRY(launch_check_finite(b->v, (long long)b->B * c.horizon * c.action_dim, b->dbg_flag, s));
    int flag = 0;
    HIP_TRY(hipMemcpy(&flag, b->dbg_flag, 4, hipMemcpyDeviceToHost));
    if (flag) return fail(RAVEL_E_STATE, "non-finite values after step " + std::to_string(b->t_host - 1));
  }
  return RAVEL_OK;
}

ravel_status ravel_step(ravel_buffer* b, const void* fop, float* action, void* stream) {
  return step_impl(b, fop, nullptr, action, stream);
}

ravel_status ravel_step_state(ravel_buffer* b, const void* fop, const float* state, float* action, void* stream) {
  if (!state) return fail(RAVEL_E_INVALID, "null state");
  return step_impl(b, fop, state, action, stream);
}

ravel_status ravel_set_relative_dims(ravel_buffer* b, const int32_t* mask) {
  if (!b) return fail(RAVEL_E_INVALID, "null buffer");
  std::lock_guard<std::mutex> lk(b->mu);
  if (b->t_host != 0) return fail(RAVEL_E_STATE, "relative dimensions must be set before the first step");
  const int D = b->m->cfg.action_dim;
  std::vector<float> mk(D, 0.f);
  bool any = false;
  for (int d = 0; mask && d < D; ++d) {
    mk[d] = mask[d] ? 1.f : 0.f;
    any = any || mask[d];
  }
  HIP_TRY(hipMemcpy(b->rel_mask, mk.data(), (size_t)D * 4, hipMemcpyHostToDevice));
  HIP_TRY(hipMemset(b->has_prev, 0, (size_t)b->B * 4));
  HIP_TRY(hipMemset(b->s_prev, 0, (size_t)b->B * D * 4));
  b->relative = any;
  return RAVEL_OK;
}

ravel_status ravel_fop_encode(ravel_buffer* b, const float* obs, void* fop_tokens, void* stream) {
  if (!b || !obs || !fop_tokens) return fail(RAVEL_E_INVALID, "null argument");
  if (!b->m->has_fop_encoder) return fail(RAVEL_E_STATE, "model has no FOP encoder weights");
  std::lock_guard<std::mutex> lk(b->mu);
  return fop_encode_impl(b, obs, fop_tokens, (hipStream_t)stream);
}

ravel_status ravel_fop_encode_noalloc(const ravel_model* mc, int32_t batch, const float* obs, void* fop_tokens,
                                      void* stream) {
  if (!mc || !obs || !fop_tokens) return fail(RAVEL_E_INVALID, "null argument");
  ravel_model* m = const_cast<ravel_model*>(mc);
  if (!m->has_fop_encoder) return fail(RAVEL_E_STATE, "model has no FOP encoder weights");
  if (batch < 1) return fail(RAVEL_E_SHAPE, "batch must be >= 1");
  const ravel_config& c = m->cfg;
  const int w = c.width, d = c.fop_obs_dim;
  int dev = 0;
  HIP_TRY(hipGetDevice(&dev));
  void* base = nullptr;
  {
    std::lock_guard<std::mutex> lk(g_scratch_mu);
    if (dev >= 0 && dev < kMaxDevices) base = g_scratch_ptr[dev];
  }
  if (!base) return fail(RAVEL_E_STATE, "no model was created on the current device (its scratch is not set up)");
  // workspace of the two GEMMs, then the staging rows, 256-byte aligned
  size_t part_elems = 0;
  int tiles = 1;
  if (m->bf16) {
    const GemmPlan p1 = plan_gemm(batch, w, d, false), p2 = plan_gemm(batch, c.n_fop * w, w, false);
    part_elems = std::max(p1.part_elems, p2.part_elems);
    tiles = std::max(std::max(p1.tiles, p2.tiles), 1);
  }
  const size_t cnt_bytes = align_up((size_t)tiles * kCounterStride * 4, 256);
  const size_t part_bytes = align_up(std::max<size_t>(part_elems, 1) * 4, 256);
  const size_t obs_bytes = align_up((size_t)batch * std::max(d, 1) * m->elt, 256);
  const size_t hid_bytes = align_up((size_t)batch * w * m->elt, 256);
  const size_t need = cnt_bytes + part_bytes + obs_bytes + hid_bytes;
  if (need > kNoAllocScratchBytes)
    return fail(RAVEL_E_INVALID, "ravel_fop_encode_noalloc: batch " + std::to_string(batch) + " needs " +
                                     std::to_string(need) + " bytes of scratch; the fixed scratch holds " +
                                     std::to_string(kNoAllocScratchBytes));
  char* q = (char*)base;
  ravel_buffer ws;  // views into the scratch only: nothing is allocated
  ws.m = m;
  ws.B = batch;
  ws.gcnt = (unsigned*)q;
  ws.gcnt_n = tiles;
  ws.gpart = (float*)(q + cnt_bytes);
  ws.gpart_elems = part_elems;
  ws.obs_t = q + cnt_bytes + part_bytes;
  ws.fhid = q + cnt_bytes + part_bytes + obs_bytes;
  hipStream_t s = (hipStream_t)stream;
  // the tickets must start at zero (an earlier call re-arms them, but a call that
  // failed half-way may not have)
  HIP_TRY(launch_zero_u32(ws.gcnt, (long long)tiles * kCounterStride, s));
  return fop_encode_impl(&ws, obs, fop_tokens, s);
}

ravel_status ravel_buffer_sync(ravel_buffer* b) {
  if (!b) return fail(RAVEL_E_INVALID, "null buffer");
  HIP_TRY(hipDeviceSynchronize());
  return check_persistent_error(b);
}

ravel_status ravel_debug_state(ravel_buffer* b, float* X_host, int64_t* t, int64_t* t_obs_host) {
  if (!b) return fail(RAVEL_E_INVALID, "null buffer");
  const ravel_config& c = b->m->cfg;
  HIP_TRY(hipDeviceSynchronize());
  RV_TRY(check_persistent_error(b));
  if (X_host) HIP_TRY(hipMemcpy(X_host, b->X, (size_t)b->B * c.horizon * c.action_dim * 4, hipMemcpyDeviceToHost));
  if (t) HIP_TRY(hipMemcpy(t, b->t, 8, hipMemcpyDeviceToHost));
  if (t_obs_host) HIP_TRY(hipMemcpy(t_obs_host, b->t_obs, (size_t)b->B * 8, hipMemcpyDeviceToHost));
  return RAVEL_OK;
}

ravel_status ravel_buffer_query(ravel_buffer* b, int32_t key, int64_t* value) {
  if (!b || !value) return fail(RAVEL_E_INVALID, "null argument");
  std::lock_guard<std::mutex> lk(b->mu);
  switch (key) {
    case RAVEL_Q_GRAPHS: *value = (int64_t)b->graphs.size(); return RAVEL_OK;
    case RAVEL_Q_PERSISTENT: *value = b->persistent ? 1 : 0; return RAVEL_OK;
    case RAVEL_Q_PHASES: *value = b->persistent ? (int64_t)b->phases.size() : 0; return RAVEL_OK;
    case RAVEL_Q_STEPS: *value = b->t_host; return RAVEL_OK;
    default: return fail(RAVEL_E_INVALID, "unknown query key");
  }
}

ravel_status ravel_publish_log(ravel_buffer* b, int64_t* entries, int32_t* n) {
  if (!b || !n) return fail(RAVEL_E_INVALID, "null argument");
  std::lock_guard<std::mutex> lk(b->mu);
  const int32_t cap = *n;
  int32_t k = 0;
  for (auto& r : b->log) {
    if (k >= cap) break;
    if (entries) {
      entries[3 * k + 0] = r[0];
      entries[3 * k + 1] = r[1];
      entries[3 * k + 2] = r[2];
    }
    ++k;
  }
  *n = entries ? k : (int32_t)b->log.size();
  return RAVEL_OK;
}

namespace {
struct BlobHeader {
  uint64_t magic;
  int32_t B, H, D, L, P, kvd, dtype, kind;
  uint64_t seed;
  int64_t t;
  int32_t relative, pad;  // relative actions: mask [D], s_prev [B, D], has_prev [B] follow the contexts
};
const uint64_t kMagic = 0x5241564C53544154ull;  // "RAVLSTAT"
}  // namespace

ravel_status ravel_buffer_save(ravel_buffer* b, void* blob, size_t* n) {
  if (!b || !n) return fail(RAVEL_E_INVALID, "null argument");
  const ravel_config& c = b->m->cfg;
  const size_t xs = (size_t)b->B * c.horizon * c.action_dim * 4;
  const size_t cs = b->ctx_elems * b->m->elt;
  const size_t rs = b->relative ? (size_t)c.action_dim * 4 + (size_t)b->B * c.action_dim * 4 + (size_t)b->B * 4 : 0;
  const size_t need = sizeof(BlobHeader) + (size_t)b->B * (8 + 4 + 4) + xs + (size_t)b->B * 2 * cs + rs;
  if (!blob) {
    *n = need;
    return RAVEL_OK;
  }
  if (*n < need) return fail(RAVEL_E_INVALID, "blob too small");
  std::lock_guard<std::mutex> lk(b->mu);
  HIP_TRY(hipDeviceSynchronize());
  char* p = (char*)blob;
  BlobHeader h{kMagic, b->B, c.horizon, c.action_dim, c.layers, c.prefix_len,
               c.n_kv_heads * c.head_dim, c.dtype, c.model_kind, b->seed, 0, b->relative ? 1 : 0, 0};
  HIP_TRY(hipMemcpy(&h.t, b->t, 8, hipMemcpyDeviceToHost));
  memcpy(p, &h, sizeof h);
  p += sizeof h;
  HIP_TRY(hipMemcpy(p, b->t_obs, (size_t)b->B * 8, hipMemcpyDeviceToHost));
  p += (size_t)b->B * 8;
  for (int e = 0; e < b->B; ++e) {
    memcpy(p, &b->active[e], 4);
    memcpy(p + 4, &b->has_ctx[e], 4);
    p += 8;
  }
  HIP_TRY(hipMemcpy(p, b->X, xs, hipMemcpyDeviceToHost));
  p += xs;
  for (int e = 0; e < b->B; ++e) {
    const size_t off = ((size_t)b->active[e] * b->B + e) * cs;
    if (cs) {
      HIP_TRY(hipMemcpy(p, (char*)b->ctx_k + off, cs, hipMemcpyDeviceToHost));
      HIP_TRY(hipMemcpy(p + cs, (char*)b->ctx_v + off, cs, hipMemcpyDeviceToHost));
    }
    p += 2 * cs;
  }
  if (b->relative) {
    const size_t D = c.action_dim;
    HIP_TRY(hipMemcpy(p, b->rel_mask, D * 4, hipMemcpyDeviceToHost));
    HIP_TRY(hipMemcpy(p + D * 4, b->s_prev, (size_t)b->B * D * 4, hipMemcpyDeviceToHost));
    HIP_TRY(hipMemcpy(p + D * 4 + (size_t)b->B * D * 4, b->has_prev, (size_t)b->B * 4, hipMemcpyDeviceToHost));
  }
  *n = need;
  return RAVEL_OK;
}

ravel_status ravel_buffer_load(ravel_buffer* b, const void* blob, size_t n) {
  if (!b || !blob) return fail(RAVEL_E_INVALID, "null argument");
  const ravel_config& c = b->m->cfg;
  const size_t xs = (size_t)b->B * c.horizon * c.action_dim * 4;
  const size_t cs = b->ctx_elems * b->m->elt;
  if (n < sizeof(BlobHeader)) return fail(RAVEL_E_INVALID, "blob too small");
  BlobHeader h;
  memcpy(&h, blob, sizeof h);
  const size_t rs = h.relative ? (size_t)c.action_dim * 4 + (size_t)b->B * c.action_dim * 4 + (size_t)b->B * 4 : 0;
  const size_t need = sizeof(BlobHeader) + (size_t)b->B * (8 + 4 + 4) + xs + (size_t)b->B * 2 * cs + rs;
  if (n < need) return fail(RAVEL_E_INVALID, "blob too small");
  if (h.magic != kMagic || h.B != b->B || h.H != c.horizon || h.D != c.action_dim || h.L != c.layers ||
      h.P != c.prefix_len || h.kvd != c.n_kv_heads * c.head_dim || h.dtype != c.dtype || h.kind != c.model_kind)
    return fail(RAVEL_E_SHAPE, "checkpoint does not match this model/batch");
  std::lock_guard<std::mutex> lk(b->mu);
  HIP_TRY(hipDeviceSynchronize());
  const char* p = (const char*)blob + sizeof h;
  b->seed = h.seed;
  HIP_TRY(hipMemcpy(b->t, &h.t, 8, hipMemcpyHostToDevice));
  b->t_host = h.t;
  HIP_TRY(hipMemcpy(b->t_obs, p, (size_t)b->B * 8, hipMemcpyHostToDevice));
  memcpy(b->tobs_host.data(), p, (size_t)b->B * 8);
  p += (size_t)b->B * 8;
  for (int e = 0; e < b->B; ++e) {
    memcpy(&b->active[e], p, 4);
    memcpy(&b->has_ctx[e], p + 4, 4);
    b->pending[e].valid = false;
    b->retire_valid[e] = 0;
    p += 8;
  }
  HIP_TRY(hipMemcpy(b->slot, b->active.data(), (size_t)b->B * 4, hipMemcpyHostToDevice));
  HIP_TRY(hipMemcpy(b->X, p, xs, hipMemcpyHostToDevice));
  p += xs;
  for (int e = 0; e < b->B; ++e) {
    const size_t off = ((size_t)b->active[e] * b->B + e) * cs;
    if (cs) {
      HIP_TRY(hipMemcpy((char*)b->ctx_k + off, p, cs, hipMemcpyHostToDevice));
      HIP_TRY(hipMemcpy((char*)b->ctx_v + off, p + cs, cs, hipMemcpyHostToDevice));
    }
    p += 2 * cs;
  }
  b->relative = h.relative != 0;
  if (b->relative) {
    const size_t D = c.action_dim;
    HIP_TRY(hipMemcpy(b->rel_mask, p, D * 4, hipMemcpyHostToDevice));
    HIP_TRY(hipMemcpy(b->s_prev, p + D * 4, (size_t)b->B * D * 4, hipMemcpyHostToDevice));
    HIP_TRY(hipMemcpy(b->has_prev, p + D * 4 + (size_t)b->B * D * 4, (size_t)b->B * 4, hipMemcpyHostToDevice));
  }
  // graphs bake in the seed as a kernel argument: rebuild them
  for (auto& g : b->graphs) {
    (void)hipGraphExecDestroy(g.exec);
    (void)hipGraphDestroy(g.graph);
  }
  b->graphs.clear();
  return RAVEL_OK;
}

ravel_status ravel_profile_step(ravel_buffer* b, const void* fop, float* action, void* stream,
                                ravel_kernel_record* records, int32_t* n) {
  if (!b || !action || !n) return fail(RAVEL_E_INVALID, "null argument");
  ravel_model* m = b->m;
  hipStream_t s = (hipStream_t)stream;
  std::lock_guard<std::mutex> lk(b->mu);
  if (m->cfg.model_kind == RAVEL_TRANSFORMER) {
    RV_TRY(apply_publishes(b, s));
    for (int e = 0; e < b->B; ++e)
      if (!b->has_ctx[e]) return fail(RAVEL_E_STATE, "env " + std::to_string(e) + " has no context yet");
  }
  if (b->relative) return fail(RAVEL_E_STATE, "profiling covers absolute actions only");
  KernelRecorder rec;
  rec.stream = s;
  ravel_status st = b->persistent ? enqueue_persistent_step(b, fop, nullptr, action, s, &rec)
                                  : enqueue_step(b, fop, nullptr, action, s, &rec);
  b->t_host += 1;
  hipError_t he = hipStreamSynchronize(s);
  const int32_t cap = *n;
  int32_t k = 0;
  for (auto& r : rec.recs) {
    if (records && k < cap) {
      ravel_kernel_record& o = records[k];
      memset(&o, 0, sizeof o);
      snprintf(o.name, sizeof o.name, "%s", r.name.c_str());
      o.bytes = r.bytes;
      o.flops = r.flops;
      (void)hipEventElapsedTime(&o.ms, r.a, r.b);
    }
    ++k;
    (void)hipEventDestroy(r.a);
    (void)hipEventDestroy(r.b);
  }
  // persistent kernel: one more record per phase class ("persistent/<class>"),
  // timed by block 0's stamps after each phase barrier; these split the
  // "persistent_layers" record and do not add to it
  if (st == RAVEL_OK && he == hipSuccess && b->persistent) {
    const size_t np = b->phases.size();
    std::vector<unsigned long long> ts(np + 1);
    int dev = 0, khz = 0;
    he = hipMemcpy(ts.data(), b->ptimes, ts.size() * sizeof(unsigned long long), hipMemcpyDeviceToHost);
    if (he == hipSuccess) he = hipGetDevice(&dev);
    if (he == hipSuccess) he = hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, dev);
    if (he == hipSuccess && khz > 0) {
      std::vector<std::string> order;
      std::map<std::string, std::array<double, 3>> agg;
      for (size_t i = 0; i < np; ++i) {
        const std::string nm = "persistent/" + b->pnames[i];
        if (!agg.count(nm)) {
          order.push_back(nm);
          agg[nm] = {0.0, 0.0, 0.0};
        }
        agg[nm][0] += (double)(ts[i + 1] - ts[i]) / (double)khz;
        agg[nm][1] += b->ph_bytes[i];
        agg[nm][2] += b->ph_flops[i];
      }
      for (auto& nm : order) {
        if (records && k < cap) {
          ravel_kernel_record& o = records[k];
          memset(&o, 0, sizeof o);
          snprintf(o.name, sizeof o.name, "%s", nm.c_str());
          o.ms = (float)agg[nm][0];
          o.bytes = agg[nm][1];
          o.flops = agg[nm][2];
        }
        ++k;
      }
      // then every phase on its own, in launch order: "phase/<index>/<class>"
      for (size_t i = 0; i < np; ++i) {
        if (records && k < cap) {
          ravel_kernel_record& o = records[k];
          memset(&o, 0, sizeof o);
          snprintf(o.name, sizeof o.name, "phase/%zu/%s", i, b->pnames[i].c_str());
          o.ms = (float)((double)(ts[i + 1] - ts[i]) / (double)khz);
          o.bytes = b->ph_bytes[i];
          o.flops = b->ph_flops[i];
        }
        ++k;
      }
    }
  }
  *n = records ? std::min(k, cap) : k;
  if (st != RAVEL_OK) return st;
  if (he != hipSuccess) return fail(RAVEL_E_HIP, hipGetErrorString(he));
  return RAVEL_OK;
}

}  // extern "C"
