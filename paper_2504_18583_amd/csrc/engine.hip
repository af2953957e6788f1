// Host side of the PARD engine: arena layout, model generation, the forward
// pass launch sequence, the speculative-decoding step and the C ABI.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "../../include/pard.h"
#include "device_init.h"
#include "pard_internal.h"

using namespace pard;

namespace {

constexpr int kPrefillRows = kMaxPassRows;   // prefill chunks run the row-block GEMM
constexpr int kDescRing = 128;
constexpr int kStepsPerPlan = 32;            // fused steps between two host checks of the length class
constexpr int kRowsSplitTarget = 224;       // workgroups a split row-block GEMM aims at (batch-32 step: 224 ahead of 192 and 256)
constexpr int kLmStrips = 8;                 // strips per lm_head workgroup at up to 16 lm rows
constexpr int kGatherMax = 4096;
constexpr size_t kRowsPartBudget = 512;   // fp32 partial tiles of split row-block GEMMs (144 KiB each)
static_assert(kRowsPartBudget * kRowsPartFloats >= kSplitPartFloats, "split partial tiles share the row-block buffer");

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }
int ceil_div(int a, int b) { return (a + b - 1) / b; }

uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}
uint64_t stream_key(uint64_t seed, uint32_t stream, uint32_t tensor) {
  return mix64((seed << 20) + ((uint64_t)stream << 16) + tensor);
}
int layer_tensor(int l, int j) { return 16 * (l + 1) + j; }

struct Bump {
  char* base = nullptr;
  size_t off = 0;
  template <class T>
  T* take(size_t count) {
    off = align256(off);
    T* p = base ? reinterpret_cast<T*>(base + off) : nullptr;
    off += count * sizeof(T);
    return p;
  }
};

// Tile plan of one skinny GEMM: S strips per workgroup, nw wavefronts splitting
// the input dimension.  nw depends only on the weight shape (for the row
// counts of decode passes), so per-element summation order does not depend on
// how many rows a pass has.
struct GemmPlan {
  int n_strips = 0, kb_total = 0;
  int nw = 4;   // one wavefront per SIMD: more waves per workgroup measured slower at every decode shape
  int ksplit = 1;   // input ranges of the skinny GEMM
};

int pick_S(int epi, int n_strips, int mt) {
  if (epi == EPI_RESID) {
    // residual GEMMs also write the per-tile row sums that the next
    // normalised GEMM adds up, so their tile count must not depend on the
    // pass: one strip per workgroup up to 256 strips (one round), two beyond
    return (n_strips > 256 && n_strips % 2 == 0) ? 2 : 1;
  }
  if (mt == 1 && epi != EPI_LOGITS) {
    // decode rows: the fewest strips per workgroup that cover the weight in
    // one round of at most 256 workgroups (one per CU), so each CU reads the
    // activation rows once; from 8 strips on the last workgroup may hold
    // fewer.  Measured (gemm_counters, 9 rows): gate/up 8B 1792 strips 7 per
    // workgroup, 37.7 us (54 at 1); Qwen2.5-7B 2368 strips 10, 43.5 us
    // against 57.1 at 2, 50.0 at 4, 56.0 at 8 and 60.5 at 9; 1B 1024 strips
    // 4, 13.7 us against 14.7 at 2 and 19.7 at 1; Qwen2.5-0.5B 608 strips 4,
    // 7.2 us against 8.1 at 2 and 9.3 at 1; QKV 8B 384 strips 2 (12.4 us
    // against 14.1 at 1), Qwen2.5-7B 288 strips 2 (12.2 against 14.8).
    for (int s : {1, 2, 4, 7, 8, 9, 10}) {
      if (s >= 7 && epi != EPI_SWIGLU) break;
      if ((s >= 8 || n_strips % s == 0) && ceil_div(n_strips, s) <= 256) return s;
    }
  }
  if (epi == EPI_SWIGLU && mt == 1) {
    // wider weights: the strips-per-workgroup count that divides the strips
    // and fills the 256 CUs most evenly; among equally even ones, the one
    // closest to two rounds of workgroups
    int best = 1, best_d = 1 << 30;
    double best_u = 0.0;
    for (int s : {7, 4, 2, 1}) {
      if (n_strips % s) continue;
      const int tiles = n_strips / s;
      const double u = (double)tiles / (ceil_div(tiles, 256) * 256);
      const int d = std::abs(tiles - 512);
      if (u > best_u + 1e-9 || (u > best_u - 1e-9 && d < best_d)) {
        best_u = u;
        best_d = d;
        best = s;
      }
    }
    return best;
  }
  int s = 1;
  // two strips share one activation stream once that still leaves >= 192
  // workgroups
  if (epi == EPI_QKV && n_strips >= 384) s = 2;
  if (epi == EPI_SWIGLU) s = 2;
  if (epi == EPI_LOGITS) s = (mt == 1) ? kLmStrips : 2;
  while (s > 1 && n_strips % s) s >>= 1;
  return s;
}

GemmPlan plan_gemm(int epi, int n_pad, int k_pad) {
  GemmPlan p;
  p.n_strips = n_pad / 16;
  p.kb_total = k_pad / 32;
  // A long, narrow residual GEMM (the 1B down projection: 128 strips x 256
  // k-blocks) fills only half the CUs with one workgroup per strip; two input
  // ranges per strip measured 11.8 against 13.6 us.  Shorter or wider shapes
  // measured slower split (the partial-tile exchange adds ~2 us of tail).
  if (epi == EPI_RESID && p.n_strips <= 128 && p.kb_total >= 256) p.ksplit = 2;
  return p;
}

// Wavefronts per workgroup for a pass of mt row tiles (LDS <= 32 KiB).
int plan_nw(const GemmPlan& p, int S, int mt) {
  int nw = p.nw;
  while (nw > 4 && nw * S * mt > 32) nw >>= 1;
  return nw;
}

// Row-block GEMM plan (passes of more than kMaxRows rows): the grid covers
// the row bound; narrow shapes split the input dimension so that about 256
// workgroups work at the typical row count, with the partial tiles in budget.
struct RowsPlan {
  int n_tiles = 0, m_blocks = 0, ksplit = 1;
};

RowsPlan plan_rows(const GemmPlan& p, int max_rows, int typ_rows) {
  RowsPlan r;
  r.n_tiles = ceil_div(p.n_strips, kRowsTileStrips);
  r.m_blocks = ceil_div(max_rows, kRowTiles * 16);
  const int live = r.n_tiles * ceil_div(std::max(1, std::min(typ_rows, max_rows)), kRowTiles * 16);
  if (live < 160) r.ksplit = ceil_div(kRowsSplitTarget, live);
  r.ksplit = std::min({r.ksplit, 16, std::max(1, p.kb_total / 8)});
  while (r.ksplit > 1 && (size_t)r.ksplit * r.n_tiles * r.m_blocks > kRowsPartBudget) --r.ksplit;
  return r;
}

// Tiles that write row sums of squares per residual GEMM (the consumers'
// ss_tiles) for passes served by the skinny or the row-block GEMM.
int resid_ss_tiles(const GemmPlan& p, bool rows) {
  return rows ? ceil_div(p.n_strips, kRowsTileStrips) * kRowsWaves : p.n_strips / pick_S(EPI_RESID, p.n_strips, 1);
}

// (max, argmax) entries per lm row.
int lm_entries(const GemmPlan& p, bool rows, int mt) {
  return rows ? ceil_div(p.n_strips, kRowsTileStrips) * kRowsWaves : p.n_strips / pick_S(EPI_LOGITS, p.n_strips, mt);
}

struct Layer {
  uint16_t *wqkv = nullptr, *wo = nullptr, *wgu = nullptr, *wd = nullptr;
  float *bqkv = nullptr, *g_attn = nullptr, *g_mlp = nullptr;
};

struct ModelDev {
  pard_model_spec spec{};
  int* ovf = nullptr;                 // fp16 range flag of this model's activations (the context's)
  int d = 0, q_dim = 0, kv_dim = 0, nqkv = 0, f_pad = 0, group = 0;
  GemmPlan p_qkv, p_o, p_gu, p_d, p_lm;
  std::vector<Layer> layers;
  uint16_t *embed = nullptr, *lm_head = nullptr;
  float* g_final = nullptr;
  uint16_t *kcache = nullptr, *vcache = nullptr;
  float2* rope = nullptr;
  float* x = nullptr;                 // residual stream, fp32 [kMaxPassRows][d]
  uint16_t* xg = nullptr;             // x * g of the next normalised GEMM (fp16, k-blocked)
  float* ss = nullptr;                // per-tile row sums of squares of x [kMaxPassRows][ss_tiles_max]
  int ss_tiles_max = 1;               // ss buffer tiles
  uint16_t *q = nullptr, *attn = nullptr, *h = nullptr;
  float* logits = nullptr;            // lm rows of the last pass [kMaxLmRows][vocab]
  int* result = nullptr;
  int2* lm_map = nullptr;             // per slot: (first lm row, lm rows) of the last pass
  FwdDesc* desc = nullptr;
};

}  // namespace

struct pard_ctx {
  ModelDev m[2];
  int mask_id = 0, max_batch = 0, max_ctx = 0, max_k = 0;
  hipStream_t stream = nullptr;
  char* arena = nullptr;
  size_t arena_bytes = 0;
  // shared device workspaces
  float* amax_val = nullptr;
  int* amax_idx = nullptr;
  float* amax_sum = nullptr;            // per-tile softmax sums (sampling)
  // speculative sampling: log2(e) / T (0: greedy) and the generator's seed
  float samp_k = 0.f;
  uint64_t samp_seed = 0;
  std::vector<int> draft_k;             // K of each slot's last granular draft pass (0: none since verify)
  float* attn_part = nullptr;
  float* rows_part = nullptr;           // also the skinny GEMM's split partial tiles
  int* split_counters = nullptr;
  SeqState* seq_dev = nullptr;
  int* out_dev = nullptr;
  size_t* gather_idx_dev = nullptr;
  float* gather_out_dev = nullptr;
  // pinned host staging
  FwdDesc* h_desc = nullptr;
  int desc_slot = 0;
  SeqState* h_seq = nullptr;
  size_t* h_gather_idx = nullptr;
  float* h_gather_out = nullptr;
  int* h_out = nullptr;
  hipEvent_t ev_start = nullptr, ev_stop = nullptr;
  // pass-boundary clock of the fused loop (device) and its host copy
  PhaseClock* clock_dev = nullptr;
  PhaseClock* h_clock = nullptr;
  double clock_khz = 0.0;
  // QKV GEMM + decode attention (+ O-projection) in one launch: one counter
  // set per layer of each model (the target's layers, then the draft's) and
  // the wait-error flag
  int* fuse_cnt = nullptr;
  int* fuse_err = nullptr;
  int* h_fuse_err = nullptr;
  bool use_fused = true;
  bool use_fused_o = true;
  bool use_fused_gu = true;
  bool use_fused_d = true;
  int gu_pre = -1, gu_pre_q = -1;   // preloaded gate/up iterations (-1: as many as the LDS holds)
  // captured fused steps (draft pass + verify pass), replayed on `stream`
  struct StepGraph { int n_seq, k, l_class; bool vsd; hipGraphExec_t exec; };
  std::vector<StepGraph> graphs;
  hipStream_t cap_stream = nullptr;     // private stream used only for capture
  bool use_graphs = true;
  // host mirrors
  std::vector<std::vector<int>> hist;   // committed tokens + pending token
  std::vector<char> prefilled;
  // per-kernel timer
  int timer_class = -1, timer_max = 0, timer_used = 0;
  std::vector<hipEvent_t> timer_ev;
  std::string err;
  size_t kv_seq_stride[2] = {0, 0};
  size_t kv_elems[2] = {0, 0};
  int kv_cap = 0;                       // KV capacity per sequence, max_ctx rounded up to 32
  int lm_rows_cap = 0;                  // lm rows of one pass
};

namespace {

pard_status fail(pard_ctx* c, pard_status s, const char* fmt, ...) {
  if (c) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    c->err = buf;
  }
  return s;
}

#define HIP_TRY(ctx, expr)                                                                  \
  do {                                                                                      \
    hipError_t e_ = (expr);                                                                 \
    if (e_ != hipSuccess)                                                                   \
      return fail((ctx), PARD_ERR_DEVICE, "%s failed: %s", #expr, hipGetErrorString(e_));   \
  } while (0)

pard_status check_spec(const pard_model_spec* s, const char* who, std::string* why) {
  char buf[256];
  auto bad = [&](pard_status st, const char* msg) {
    snprintf(buf, sizeof buf, "%s spec: %s", who, msg);
    *why = buf;
    return st;
  };
  if (!s) return bad(PARD_ERR_ARG, "null");
  if (s->n_layers < 1 || s->n_layers > 4000) return bad(PARD_ERR_ARG, "n_layers out of range");
  if (s->d_model < 32 || s->n_heads < 1 || s->n_kv_heads < 1 || s->ffn_dim < 1 || s->vocab < 16)
    return bad(PARD_ERR_ARG, "non-positive dimension");
  if (s->n_heads % s->n_kv_heads) return bad(PARD_ERR_ARG, "n_heads not a multiple of n_kv_heads");
  if (!(s->rms_eps > 0.f) || !(s->rope_theta > 1.f) || !(s->init_std > 0.f))
    return bad(PARD_ERR_ARG, "rms_eps, rope_theta or init_std out of range");
  if (s->rope_factor != 0.f &&
      (!(s->rope_factor >= 1.f) || !std::isfinite(s->rope_factor) || !(s->rope_low_freq_factor > 0.f) ||
       !(s->rope_high_freq_factor > s->rope_low_freq_factor) || !std::isfinite(s->rope_high_freq_factor) ||
       s->rope_original_max_pos < 1))
    return bad(PARD_ERR_ARG, "rope scaling: need factor >= 1, 0 < low < high, original length >= 1");
  if (s->seed >= (1ull << 44) || s->weight_stream >= 16) return bad(PARD_ERR_ARG, "seed or weight_stream out of range");
  if (s->dtype != PARD_BF16) return bad(PARD_ERR_UNSUPPORTED, "only bf16 weights are supported");
  if (s->head_dim != 64 && s->head_dim != 128) return bad(PARD_ERR_UNSUPPORTED, "head_dim must be 64 or 128");
  if (s->d_model % 32) return bad(PARD_ERR_UNSUPPORTED, "d_model must be a multiple of 32");
  if (s->vocab % 16) return bad(PARD_ERR_UNSUPPORTED, "vocab must be a multiple of 16");
  if ((int64_t)s->vocab * s->d_model >= (1ll << 40)) return bad(PARD_ERR_ARG, "vocab too large");
  // every strip-packed matrix is addressed with 32-bit byte offsets (buffer
  // descriptors, k-block offsets): rows padded to 16, columns to 32, 2 bytes each
  auto pad = [](int64_t v, int64_t m) { return (v + m - 1) / m * m; };
  const int64_t d = s->d_model, q = (int64_t)s->n_heads * s->head_dim, kv = (int64_t)s->n_kv_heads * s->head_dim;
  const int64_t f = pad(s->ffn_dim, 32);
  const int64_t mats[5][2] = {{q + 2 * kv, d}, {d, q}, {2 * f, d}, {d, f}, {s->vocab, d}};
  for (const auto& m : mats)
    if (pad(m[0], 16) * pad(m[1], 32) * 2 >= (1ll << 31))
      return bad(PARD_ERR_UNSUPPORTED, "a weight matrix reaches 2 GiB (32-bit byte offsets)");
  return PARD_OK;
}

pard_status check_all(const pard_model_spec* t, const pard_model_spec* d, int mask_id, int max_batch,
                      int max_ctx, int max_k, std::string* why) {
  pard_status st = check_spec(t, "target", why);
  if (st != PARD_OK) return st;
  st = check_spec(d, "draft", why);
  if (st != PARD_OK) return st;
  if (t->vocab != d->vocab) { *why = "target and draft vocab differ"; return PARD_ERR_ARG; }
  if (mask_id < 0 || mask_id >= t->vocab) { *why = "mask_id out of range"; return PARD_ERR_ARG; }
  if (max_k < 1 || max_k > kMaxK) { *why = "max_k must be in [1, 32]"; return PARD_ERR_ARG; }
  if (max_batch < 1 || max_batch > 4096) { *why = "max_batch out of range"; return PARD_ERR_ARG; }
  if (max_ctx < 2 * max_k + 2 || max_ctx > (1 << 24)) { *why = "max_ctx out of range"; return PARD_ERR_ARG; }
  return PARD_OK;
}

void derive(ModelDev& M, const pard_model_spec& s, int max_ctx) {
  M.spec = s;
  M.d = s.d_model;
  M.q_dim = s.n_heads * s.head_dim;
  M.kv_dim = s.n_kv_heads * s.head_dim;
  M.nqkv = M.q_dim + 2 * M.kv_dim;
  M.f_pad = ceil_div(s.ffn_dim, 32) * 32;
  M.group = s.n_heads / s.n_kv_heads;
  M.p_qkv = plan_gemm(EPI_QKV, M.nqkv, M.d);
  M.p_o = plan_gemm(EPI_RESID, M.d, M.q_dim);
  // one strip per workgroup: eight wavefronts over the input (at every row
  // tile count), as the O units fused into the QKV + attention launch use,
  // so a row's O-projection is summed in the same order whether or not its
  // pass runs fused (the unfused launch measured 8.3 -> 10.9 us at the 8B
  // shape for it; 16k-context 8B/1B step 4.53 -> 4.57 ms)
  if (pick_S(EPI_RESID, M.p_o.n_strips, 1) == 1) M.p_o.nw = 8;
  M.p_gu = plan_gemm(EPI_SWIGLU, 2 * M.f_pad, M.d);
  M.p_d = plan_gemm(EPI_RESID, M.d, M.f_pad);
  M.p_lm = plan_gemm(EPI_LOGITS, s.vocab, M.d);
  M.ss_tiles_max = std::max(resid_ss_tiles(M.p_o, false), resid_ss_tiles(M.p_o, true));
}

// Lays out (base == nullptr: sizes) every device region of a context.
size_t layout(pard_ctx* c, char* base) {
  Bump b;
  b.base = base;
  int max_lm_tiles = 1;
  // lm rows of one pass: K + 1 per sequence of a batched step (or a prefill row)
  const int lm_rows_cap = std::min(kMaxLmRows, std::min(c->max_batch, kMaxPassSeqs) * (c->max_k + 1));
  c->lm_rows_cap = lm_rows_cap;
  size_t attn_part = 1;
  const int cap = c->kv_cap;
  for (int w = 0; w < 2; ++w) {
    ModelDev& M = c->m[w];
    const pard_model_spec& s = M.spec;
    M.layers.assign(s.n_layers, Layer{});
    for (int l = 0; l < s.n_layers; ++l) {
      Layer& L = M.layers[l];
      L.wqkv = b.take<uint16_t>((size_t)M.nqkv * M.d);
      L.wo = b.take<uint16_t>((size_t)M.d * M.q_dim);
      L.wgu = b.take<uint16_t>((size_t)2 * M.f_pad * M.d);
      L.wd = b.take<uint16_t>((size_t)M.d * M.f_pad);
      L.bqkv = s.qkv_bias ? b.take<float>(M.nqkv) : nullptr;
      L.g_attn = b.take<float>(M.d);
      L.g_mlp = b.take<float>(M.d);
    }
    M.embed = b.take<uint16_t>((size_t)s.vocab * M.d);
    M.lm_head = s.tied_embeddings ? M.embed : b.take<uint16_t>((size_t)s.vocab * M.d);
    M.g_final = b.take<float>(M.d);
    const size_t kv = (size_t)c->max_batch * s.n_layers * s.n_kv_heads * cap * s.head_dim;
    c->kv_seq_stride[w] = (size_t)s.n_layers * s.n_kv_heads * cap * s.head_dim;
    c->kv_elems[w] = kv;
    M.kcache = b.take<uint16_t>(kv);
    M.vcache = b.take<uint16_t>(kv);
    M.rope = b.take<float2>((size_t)cap * s.head_dim / 2);
    M.x = b.take<float>((size_t)kMaxPassRows * M.d);
    M.xg = b.take<uint16_t>((size_t)kMaxPassRows * M.d);
    M.ss = b.take<float>((size_t)std::max(1, M.ss_tiles_max) * kMaxPassRows);
    M.q = b.take<uint16_t>((size_t)kMaxPassRows * M.q_dim);
    M.attn = b.take<uint16_t>((size_t)kMaxPassRows * M.q_dim);
    M.h = b.take<uint16_t>((size_t)kMaxPassRows * M.f_pad);
    M.logits = b.take<float>((size_t)lm_rows_cap * s.vocab);
    M.result = b.take<int>(kMaxLmRows);
    M.lm_map = b.take<int2>(c->max_batch);
    M.desc = b.take<FwdDesc>(1);
    max_lm_tiles = std::max(max_lm_tiles, M.p_lm.n_strips);
    attn_part = std::max(attn_part, (size_t)s.n_kv_heads * kAttnRecords *
                                        attn_part_floats(s.head_dim, attn_max_q_tiles(s.head_dim)));
  }
  c->amax_val = b.take<float>((size_t)max_lm_tiles * lm_rows_cap);
  c->amax_idx = b.take<int>((size_t)max_lm_tiles * lm_rows_cap);
  c->amax_sum = b.take<float>((size_t)max_lm_tiles * lm_rows_cap);
  c->attn_part = b.take<float>(attn_part);
  c->rows_part = b.take<float>(kRowsPartBudget * kRowsPartFloats);
  c->split_counters = b.take<int>(kSplitCounters);
  c->seq_dev = b.take<SeqState>(c->max_batch);
  c->out_dev = b.take<int>((size_t)c->max_batch * c->max_ctx);
  c->gather_idx_dev = b.take<size_t>(kGatherMax);
  c->gather_out_dev = b.take<float>(kGatherMax);
  c->clock_dev = b.take<PhaseClock>(1);
  c->fuse_cnt = b.take<int>((size_t)kFuseInts * (c->m[0].spec.n_layers + c->m[1].spec.n_layers));
  c->fuse_err = b.take<int>(64);
  // ints 0: a fused launch's wait gave up; 32: an fp16 activation overflowed
  c->m[0].ovf = c->m[1].ovf = c->fuse_err ? c->fuse_err + 32 : nullptr;
  return align256(b.off);
}

// ----------------------------------------------------------------------------
// weight generation
// ----------------------------------------------------------------------------

pard_status generate(pard_ctx* c, int w) {
  ModelDev& M = c->m[w];
  const pard_model_spec& s = M.spec;
  const double stdv = s.init_std;
  auto key = [&](int tensor) { return stream_key(s.seed, s.weight_stream, (uint32_t)tensor); };
  auto gen = [&](uint16_t* dst, int n_pad, int k_pad, int rows, int cols, int map, uint64_t k0, uint64_t k1,
                 uint64_t k2) -> hipError_t {
    GenArgs a{};
    a.dst = dst;
    a.n_strips = n_pad / 16;
    a.kb_total = k_pad / 32;
    a.rows = rows;
    a.cols = cols;
    a.map = map;
    a.q_dim = M.q_dim;
    a.kv_dim = M.kv_dim;
    a.hd = s.head_dim;
    a.key0 = k0;
    a.key1 = k1;
    a.key2 = k2;
    a.stdv = stdv;
    return launch_gen_packed(a, c->stream);
  };
  for (int l = 0; l < s.n_layers; ++l) {
    Layer& L = M.layers[l];
    HIP_TRY(c, gen(L.wqkv, M.nqkv, M.d, 0, M.d, MAP_QKV, key(layer_tensor(l, 0)), key(layer_tensor(l, 1)),
                   key(layer_tensor(l, 2))));
    HIP_TRY(c, gen(L.wo, M.d, M.q_dim, M.d, M.q_dim, MAP_IDENTITY, key(layer_tensor(l, 3)), 0, 0));
    HIP_TRY(c, gen(L.wgu, 2 * M.f_pad, M.d, s.ffn_dim, M.d, MAP_GATEUP, key(layer_tensor(l, 4)),
                   key(layer_tensor(l, 5)), 0));
    HIP_TRY(c, gen(L.wd, M.d, M.f_pad, M.d, s.ffn_dim, MAP_IDENTITY, key(layer_tensor(l, 6)), 0, 0));
    if (L.bqkv) {
      GenArgs a{};
      a.map = MAP_QKV;
      a.q_dim = M.q_dim;
      a.kv_dim = M.kv_dim;
      a.hd = s.head_dim;
      a.key0 = key(layer_tensor(l, 7));
      a.key1 = key(layer_tensor(l, 8));
      a.key2 = key(layer_tensor(l, 9));
      a.stdv = stdv;
      HIP_TRY(c, launch_gen_bias(a, L.bqkv, M.nqkv, c->stream));
    }
    HIP_TRY(c, launch_fill_f32(L.g_attn, M.d, 1.0f, c->stream));
    HIP_TRY(c, launch_fill_f32(L.g_mlp, M.d, 1.0f, c->stream));
  }
  HIP_TRY(c, gen(M.embed, s.vocab, M.d, s.vocab, M.d, MAP_IDENTITY, key(0), 0, 0));
  if (!s.tied_embeddings) HIP_TRY(c, gen(M.lm_head, s.vocab, M.d, s.vocab, M.d, MAP_IDENTITY, key(1), 0, 0));
  HIP_TRY(c, launch_fill_f32(M.g_final, M.d, 1.0f, c->stream));
  RopeScaling sc;
  if (s.rope_factor != 0.f) {
    sc.factor = s.rope_factor;
    sc.low = s.rope_low_freq_factor;
    sc.high = s.rope_high_freq_factor;
    sc.orig = s.rope_original_max_pos;
  }
  HIP_TRY(c, launch_rope_table(M.rope, c->kv_cap, s.head_dim, (double)s.rope_theta, sc, c->stream));
  // zero KV caches: padded key tiles read stale slots, which must hold finite values
  HIP_TRY(c, launch_fill_u32(reinterpret_cast<uint32_t*>(M.kcache), c->kv_elems[w] / 2, 0u, c->stream));
  HIP_TRY(c, launch_fill_u32(reinterpret_cast<uint32_t*>(M.vcache), c->kv_elems[w] / 2, 0u, c->stream));
  return PARD_OK;
}

// ----------------------------------------------------------------------------
// forward pass
// ----------------------------------------------------------------------------

struct Timed {
  pard_ctx* c;
  bool on;
  Timed(pard_ctx* ctx, int cls) : c(ctx), on(false) {
    if (c->timer_class == cls && c->timer_used < c->timer_max) {
      on = hipEventRecord(c->timer_ev[2 * c->timer_used], c->stream) == hipSuccess;
    }
  }
  ~Timed() {
    if (on) {
      (void)hipEventRecord(c->timer_ev[2 * c->timer_used + 1], c->stream);
      ++c->timer_used;
    }
  }
};

GemmArgs gemm_base(const ModelDev& M, const uint16_t* W, int act_rows) {
  GemmArgs a{};
  a.W = W;
  a.act_rows = act_rows;
  a.desc = M.desc;
  a.eps = M.spec.rms_eps;
  a.inv_k = 1.0f / (float)M.d;
  a.ss_stride = std::max(1, M.ss_tiles_max);
  a.ovf = M.ovf;
  return a;
}

// The fused launches' counter sets of model w (one per layer).
int* fuse_counters(pard_ctx* c, int w) {
  return c->fuse_cnt + (w == 0 ? 0 : (size_t)kFuseInts * c->m[0].spec.n_layers);
}

// O-projection + residual: x += attn W_o^T, then fp16(x * g_mlp) and the row
// sums of squares for the gate/up GEMM.
GemmArgs o_args(const ModelDev& M, const Layer& L, int act_rows) {
  GemmArgs a = gemm_base(M, L.wo, act_rows);
  a.A = M.attn;
  a.lda = M.q_dim;
  a.x = M.x;
  a.ldx = M.d;
  a.g_next = L.g_mlp;
  a.xg = M.xg;
  a.ss_out = M.ss;
  a.kb_total = M.p_o.kb_total;
  a.n_strips = M.p_o.n_strips;
  a.n_tiles = M.p_o.n_strips;
  a.ksplit = 1;
  a.kb_split = M.p_o.kb_total;
  return a;
}

// Norm + gate/up + SiLU * up: h = silu(x g W_gate^T / rms) * (x g W_up^T / rms).
// S > 0: the tile plan of a fused launch (S strips per tile, one input range).
GemmArgs gu_args(const ModelDev& M, const Layer& L, int act_rows, int ss_tiles, int S) {
  GemmArgs a = gemm_base(M, L.wgu, act_rows);
  a.A = M.xg;
  a.lda = M.d;
  a.ss_in = M.ss;
  a.ss_tiles = ss_tiles;
  a.out = M.h;
  if (S > 0) {
    a.kb_total = M.p_gu.kb_total;
    a.n_strips = M.p_gu.n_strips;
    a.n_tiles = M.p_gu.n_strips / S;
    a.ksplit = 1;
    a.kb_split = M.p_gu.kb_total;
  }
  return a;
}

// Down projection + residual of layer l: x += h W_down^T, then fp16(x * g)
// for the next layer's (or the final) norm and the row sums of squares.
// fused: the tile plan of a fused launch (one strip per tile, the plan's
// input ranges; part and counters for the partial-tile exchange).
GemmArgs d_args(const ModelDev& M, int l, int act_rows, bool fused, float* part, int* counters) {
  GemmArgs a = gemm_base(M, M.layers[l].wd, act_rows);
  a.A = M.h;
  a.lda = M.f_pad;
  a.x = M.x;
  a.ldx = M.d;
  a.g_next = (l + 1 < M.spec.n_layers) ? M.layers[l + 1].g_attn : M.g_final;
  a.xg = M.xg;
  a.ss_out = M.ss;
  if (fused) {
    a.kb_total = M.p_d.kb_total;
    a.n_strips = M.p_d.n_strips;
    a.n_tiles = M.p_d.n_strips;
    a.ksplit = M.p_d.ksplit;
    a.kb_split = ceil_div(M.p_d.kb_total, M.p_d.ksplit);
    a.part = part;
    a.counters = counters;
  }
  return a;
}

struct PassSpec {
  int max_rows = 1;       // upper bound of n_rows (sets the M tiles)
  int typ_rows = 0;       // row count the split plan is tuned for (0: max_rows)
  int max_lm_rows = 0;    // 0: no lm_head
  int n_seq = 1;          // upper bound of the pass's sequences
  int max_seq_rows = 0;   // upper bound of one sequence's rows (0: max_rows)
  int l_bound = 0;        // upper bound of pos0 + n_rows (attention split plan)
  int tail = TAIL_NONE;
  FwdDesc* next_desc = nullptr;
  bool emit = false;
};

// One GEMM of a pass: the skinny kernel up to kMaxRows rows, the row-block
// kernel above.
hipError_t run_gemm(pard_ctx* c, int cls, int epi, int max_rows, int typ_rows, GemmArgs a, const GemmPlan& p) {
  // a timed GEMM launch carries its events: they take the kernel's own start
  // and end timestamps, not those of separate marker packets
  LaunchEvents ev;
  if (c->timer_class == cls && c->timer_used < c->timer_max) {
    ev.start = c->timer_ev[2 * c->timer_used];
    ev.stop = c->timer_ev[2 * c->timer_used + 1];
    ++c->timer_used;
  }
  a.kb_total = p.kb_total;
  a.n_strips = p.n_strips;
  if (max_rows > kMaxRows) {
    const RowsPlan r = plan_rows(p, max_rows, typ_rows > 0 ? typ_rows : max_rows);
    a.n_tiles = r.n_tiles;
    a.m_blocks = r.m_blocks;
    a.ksplit = r.ksplit;
    a.part = c->rows_part;
    return launch_gemm_rows(epi, a, c->stream, ev);
  }
  const int mt = ceil_div(max_rows, 16);
  const int S = pick_S(epi, p.n_strips, mt);
  a.n_tiles = ceil_div(p.n_strips, S);
  a.ksplit = p.ksplit;
  a.kb_split = ceil_div(p.kb_total, p.ksplit);
  a.part = c->rows_part;
  a.counters = c->split_counters;
  return launch_gemm(epi, mt, S, plan_nw(p, S, mt), a, c->stream, ev);
}

pard_status forward(pard_ctx* c, int w, const PassSpec& ps) {
  ModelDev& M = c->m[w];
  const pard_model_spec& s = M.spec;
  const bool rows = ps.max_rows > kMaxRows;
  const int typ = ps.typ_rows > 0 ? ps.typ_rows : ps.max_rows;
  const int ss_tiles = resid_ss_tiles(M.p_o, rows);
  const int act_rows = rows ? kMaxPassRows : kMaxRows;
  const int cls0 = w * 8;
  if (ps.max_rows < 1 || ps.max_rows > kMaxPassRows || ps.n_seq < 1 || ps.n_seq > kMaxPassSeqs ||
      ps.max_lm_rows > c->lm_rows_cap)
    return fail(c, PARD_ERR_CAPACITY, "pass of %d rows / %d sequences exceeds the engine's limits", ps.max_rows,
                ps.n_seq);
  {
    Timed t(c, cls0 + 0);
    HIP_TRY(c, launch_embed(M.embed, M.p_lm.n_strips, M.d, M.desc, M.x, M.layers[0].g_attn, M.xg, act_rows, M.ss,
                            std::max(1, M.ss_tiles_max), ps.max_rows, &c->clock_dev->pass_start[w],
                            fuse_counters(c, w), s.n_layers, M.ovf, c->stream));
  }
  const size_t layer_kv = (size_t)s.n_kv_heads * c->kv_cap * s.head_dim;
  // attention plan: one workgroup per (sequence, KV head, query group, key
  // chunk); a query group holds every (row, head) pair of the KV head for
  // decode passes (up to 48 / 64 pairs); chunks start at fixed multiples of
  // the chunk length, which depends only on the pass's shape and context
  // bound, never on its rows' contents (kAttnChunk keys; decode passes over
  // long contexts and very long prefill chunks use longer ones)
  const int seq_rows = ps.max_seq_rows > 0 ? std::min(ps.max_seq_rows, ps.max_rows) : ps.max_rows;
  const int qpairs = seq_rows * M.group;
  const int l_bound = std::min(std::max(ps.l_bound, 1), c->kv_cap);
  // decode passes over a short context: one chunk per workgroup of 8 waves
  // (no merge kernel), one query tile per workgroup (at head_dim 128 that keeps
  // the 8-wave kernel within its registers; at 64 it measured fastest)
  const bool wide = !rows && l_bound <= kAttnWideMaxKeys;
  int nqt = std::min(attn_max_q_tiles(s.head_dim), ceil_div(qpairs, 16));
  if (wide) nqt = std::min(nqt, s.head_dim == 128 ? 1 : kAttnWideQTiles64);
  const int n_qblocks = ceil_div(qpairs, 16 * nqt);
  if (ps.n_seq * n_qblocks > kAttnRecords)
    return fail(c, PARD_ERR_CAPACITY, "attention plan: %d query blocks exceed the record budget", ps.n_seq * n_qblocks);
  int split_len = wide ? ceil_div(l_bound, 128) * 128 : kAttnChunk;
  // row-block passes over several sequences (batched decode): 1024-key
  // chunks (batch-32 step 15.5 ms with 256, 15.4 with 512, 15.2 with 1024;
  // whole contexts, up to 2048 keys, 16.3)
  if (rows && ps.n_seq > 1) split_len = kAttnBatchChunk;
  // decode passes over long contexts and single-sequence prefill chunks: the
  // shortest chunk (a multiple of 128 keys) that keeps the grid within one
  // workgroup per CU (16k keys, 8B/1B step: 5.33 ms with 256-key chunks, 5.06
  // with 1024, 4.91 with 640; 16k-token prefill 839 -> 807 ms)
  if (!wide && (!rows || ps.n_seq == 1)) {
    const int per = std::max(1, kAttnDecodeWGs / (ps.n_seq * s.n_kv_heads * n_qblocks));
    split_len = std::min(kAttnLongChunkMax, std::max(split_len, ceil_div(ceil_div(l_bound, per), 128) * 128));
  }
  while ((int64_t)ps.n_seq * n_qblocks * ceil_div(l_bound, split_len) > kAttnRecords) split_len *= 2;
  const int n_splits = ceil_div(l_bound, split_len);
  // decode passes over one attention chunk: QKV GEMM and attention in one
  // launch when its grid fits the device at once
  const int mt_q = ceil_div(ps.max_rows, 16);
  const int S_q = rows ? 0 : pick_S(EPI_QKV, M.p_qkv.n_strips, mt_q);
  const int n_attn_wg = s.n_kv_heads * n_qblocks * ps.n_seq;
  const bool fused = c->use_fused && !rows && wide && nqt == 1 && M.p_qkv.ksplit == 1 && S_q > 0 &&
                     M.p_qkv.n_strips % S_q == 0 &&
                     M.p_qkv.n_strips / S_q + n_attn_wg <= qkv_attn_capacity(mt_q, S_q, s.head_dim);
  // one row tile: the O-projection joins the launch too, its weights
  // streaming while the attention runs.  Workers are the QKV workgroups plus
  // extra ones in the room the device has left; the extras start with the
  // launch and take two units where the strips outnumber the workers.  The
  // units sum over eight wavefronts, as the unfused O-projection does.
  FuseCtl fo;
  bool fused_o = false;
  if (fused && c->use_fused_o && mt_q == 1 && M.p_o.ksplit == 1 && M.p_o.nw == 8) {
    const int n_qkv = M.p_qkv.n_strips / S_q;
    const int cap = qkv_attn_capacity(1, S_q, s.head_dim, M.p_o.kb_total);
    const int room = cap - n_qkv - n_attn_wg;
    fo.o_units = M.p_o.n_strips;
    fo.o_extra = std::max(0, std::min(room, fo.o_units - n_qkv));
    fo.o_two = std::max(0, fo.o_units - n_qkv - fo.o_extra);
    fused_o = cap > 0 && room >= 0 && fo.o_two <= fo.o_extra;
  }
  // with O units, the gate/up GEMM joins as well: every workgroup of the grid
  // runs one gate/up tile, whose first weight blocks it loads into LDS while
  // the attention runs (extras are added until the grid covers the tiles)
  const int S_gu = pick_S(EPI_SWIGLU, M.p_gu.n_strips, 1);
  bool fused_gu = false, fused_d = false;
  if (fused_o && c->use_fused_gu && (S_gu == 4 || S_gu == 7) && M.p_gu.ksplit == 1 &&
      M.p_gu.n_strips % S_gu == 0 && plan_nw(M.p_gu, S_gu, 1) == 4) {
    const int n_qkv = M.p_qkv.n_strips / S_q;
    const int gu_tiles = M.p_gu.n_strips / S_gu;
    // and the down projection (one strip per tile, one input range), whose
    // workgroups wait for every gate/up tile
    const int d_S = c->use_fused_d && M.p_d.ksplit <= 2 && pick_S(EPI_RESID, M.p_d.n_strips, 1) == 1 &&
                    plan_nw(M.p_d, 1, 1) == 4 ? 1 : 0;
    const int d_units = d_S ? M.p_d.n_strips * M.p_d.ksplit : 0;
    const int pre_max = std::min(qkv_attn_gu_pre_max(S_q, s.head_dim, M.p_o.kb_total, S_gu, d_S), M.p_gu.kb_total / 4);
    const int pre = c->gu_pre >= 0 ? std::min(c->gu_pre, pre_max) : pre_max;
    const int pre_q = c->gu_pre_q >= 0 ? std::min(c->gu_pre_q, pre) : pre;
    const int cap = pre >= 1 ? qkv_attn_capacity(1, S_q, s.head_dim, M.p_o.kb_total, S_gu, pre, d_S) : 0;
    FuseCtl t = fo;
    t.o_extra = std::max({fo.o_extra, gu_tiles - n_qkv - n_attn_wg, d_units - n_qkv - n_attn_wg});
    t.o_two = std::max(0, t.o_units - n_qkv - t.o_extra);
    if (cap > 0 && gu_tiles <= cap && n_qkv + n_attn_wg + t.o_extra <= cap && t.o_two <= t.o_extra) {
      fused_gu = true;
      fused_d = d_S == 1;
      t.gu_tiles = gu_tiles;
      t.gu_pre = pre;
      t.gu_pre_q = pre_q;
      t.n_odone = std::min(n_qkv + t.o_extra, t.o_units - t.o_two);
      t.d_tiles = d_units;
      fo = t;
    }
  }
  for (int l = 0; l < s.n_layers; ++l) {
    const Layer& L = M.layers[l];
    uint16_t* kc = M.kcache + layer_kv * l;
    uint16_t* vc = M.vcache + layer_kv * l;
    AttnArgs aa{};
    aa.q = M.q;
    aa.ldq = M.q_dim;
    aa.kc = kc;
    aa.vc = vc;
    aa.kv_seq_stride = c->kv_seq_stride[w];
    aa.cap = c->kv_cap;
    aa.out = M.attn;
    aa.act_rows = act_rows;
    aa.desc = M.desc;
    aa.n_heads = s.n_heads;
    aa.n_kv = s.n_kv_heads;
    aa.nqt = nqt;
    aa.n_qblocks = n_qblocks;
    aa.split_len = split_len;
    aa.n_splits = n_splits;
    aa.n_seq = ps.n_seq;
    aa.scale = 1.0f / std::sqrt((float)s.head_dim);
    aa.part = c->attn_part;
    aa.wide = wide ? 1 : 0;
    {  // norm + QKV + bias + RoPE + KV append (and, fused, the attention)
      GemmArgs a = gemm_base(M, L.wqkv, act_rows);
      a.A = M.xg;
      a.lda = M.d;
      a.ss_in = M.ss;
      a.ss_tiles = l == 0 ? 1 : ss_tiles;
      a.out = M.q;
      a.ld_out = M.q_dim;
      a.kc = kc;
      a.vc = vc;
      a.cap = c->kv_cap;
      a.kv_seq_stride = c->kv_seq_stride[w];
      a.bias = L.bqkv;
      a.rope = M.rope;
      a.q_dim = M.q_dim;
      a.kv_dim = M.kv_dim;
      a.hd = s.head_dim;
      if (fused) {
        a.kb_total = M.p_qkv.kb_total;
        a.n_strips = M.p_qkv.n_strips;
        a.n_tiles = M.p_qkv.n_strips / S_q;
        a.ksplit = 1;
        a.kb_split = M.p_qkv.kb_total;
        FuseCtl f = fused_o ? fo : FuseCtl{};
        f.counters = fuse_counters(c, w) + (size_t)l * kFuseInts;
        f.err = c->fuse_err;
        f.n_prod = a.n_tiles;
        f.n_cons = n_attn_wg;
        GemmArgs o{}, gu{}, dn{};
        if (fused_o) o = o_args(M, L, act_rows);
        if (fused_gu) gu = gu_args(M, L, act_rows, ss_tiles, S_gu);
        if (fused_d) dn = d_args(M, l, act_rows, true, c->rows_part, c->split_counters);
        // the kernel timer's QKV class covers the fused launch (attention included)
        LaunchEvents ev;
        if (c->timer_class == cls0 + 1 && c->timer_used < c->timer_max) {
          ev.start = c->timer_ev[2 * c->timer_used];
          ev.stop = c->timer_ev[2 * c->timer_used + 1];
          ++c->timer_used;
        }
        HIP_TRY(c, launch_qkv_attn(mt_q, S_q, s.head_dim, a, aa, f, fused_o ? &o : nullptr, fused_gu ? &gu : nullptr,
                                   S_gu, fused_d ? &dn : nullptr, c->stream, ev));
      } else {
        HIP_TRY(c, run_gemm(c, cls0 + 1, EPI_QKV, ps.max_rows, typ, a, M.p_qkv));
      }
    }
    if (!fused) {  // attention
      Timed t(c, cls0 + 2);
      HIP_TRY(c, launch_attention(s.head_dim, aa, c->stream));
    }
    if (!fused_o) {  // O-projection + residual
      HIP_TRY(c, run_gemm(c, cls0 + 3, EPI_RESID, ps.max_rows, typ, o_args(M, L, act_rows), M.p_o));
    }
    if (!fused_gu) {  // norm + gate/up + SiLU * up
      HIP_TRY(c, run_gemm(c, cls0 + 4, EPI_SWIGLU, ps.max_rows, typ, gu_args(M, L, act_rows, ss_tiles, 0), M.p_gu));
    }
    if (!fused_d) {  // down + residual
      HIP_TRY(c, run_gemm(c, cls0 + 5, EPI_RESID, ps.max_rows, typ, d_args(M, l, act_rows, false, nullptr, nullptr),
                          M.p_d));
    }
  }
  if (ps.max_lm_rows > 0) {
    const bool lm_rows = ps.max_lm_rows > kMaxRows;
    const int mt_lm = ceil_div(ps.max_lm_rows, 16);
    GemmArgs a = gemm_base(M, M.lm_head, act_rows);
    a.A = M.xg;
    a.lda = M.d;
    a.ss_in = M.ss;
    a.ss_tiles = ss_tiles;
    a.logits = M.logits;
    a.vocab = s.vocab;
    a.amax_val = c->amax_val;
    a.amax_idx = c->amax_idx;
    a.amax_stride = lm_entries(M.p_lm, lm_rows, mt_lm);
    a.samp_k = c->samp_k;
    a.amax_sum = c->amax_sum;
    HIP_TRY(c, run_gemm(c, cls0 + 6, EPI_LOGITS, ps.max_lm_rows, ps.max_lm_rows, a, M.p_lm));
    TailArgs ta{};
    ta.desc = M.desc;
    ta.amax_val = c->amax_val;
    ta.amax_idx = c->amax_idx;
    ta.n_tiles = a.amax_stride;
    ta.vocab = s.vocab;
    ta.result = M.result;
    ta.tail = ps.tail;
    ta.states = c->seq_dev;
    ta.lm_map = M.lm_map;
    ta.lm_map_draft = c->m[PARD_DRAFT].lm_map;
    ta.next_desc = ps.next_desc;
    ta.out_tokens = ps.emit ? c->out_dev : nullptr;
    ta.out_cap = c->max_ctx;
    ta.samp_k = c->samp_k;
    ta.seed = c->samp_seed;
    ta.amax_sum = c->amax_sum;
    ta.logits = M.logits;
    ta.q_logits = c->m[PARD_DRAFT].logits;
    ta.tile_w = lm_rows ? kRowsWaveStrips * 16 : pick_S(EPI_LOGITS, M.p_lm.n_strips, mt_lm) * 16;
    ta.clock = c->clock_dev;
    Timed t(c, cls0 + 7);
    HIP_TRY(c, launch_tail(ta, ps.n_seq, c->stream));
    if (ps.n_seq > 1 && ps.next_desc) HIP_TRY(c, launch_stage(ta, c->stream));
  }
  return PARD_OK;
}

// Copies a host-built pass description into model w's device descriptor.
pard_status stage_desc(pard_ctx* c, int w, const FwdDesc& d) {
  if (c->desc_slot == kDescRing) {
    HIP_TRY(c, hipStreamSynchronize(c->stream));
    c->desc_slot = 0;
  }
  FwdDesc* h = c->h_desc + c->desc_slot++;
  *h = d;
  HIP_TRY(c, hipMemcpyAsync(c->m[w].desc, h, sizeof(FwdDesc), hipMemcpyHostToDevice, c->stream));
  return PARD_OK;
}

pard_status push_seq(pard_ctx* c, int seq) {
  HIP_TRY(c, hipMemcpyAsync(c->seq_dev + seq, c->h_seq + seq, sizeof(SeqState), hipMemcpyHostToDevice, c->stream));
  return PARD_OK;
}

pard_status pull_seqs_sync(pard_ctx* c, const int* seqs, int n) {
  for (int i = 0; i < n; ++i)
    HIP_TRY(c, hipMemcpyAsync(c->h_seq + seqs[i], c->seq_dev + seqs[i], sizeof(SeqState), hipMemcpyDeviceToHost,
                              c->stream));
  HIP_TRY(c, hipMemcpyAsync(c->h_fuse_err, c->fuse_err, sizeof(int) * 64, hipMemcpyDeviceToHost, c->stream));
  HIP_TRY(c, hipStreamSynchronize(c->stream));
  c->desc_slot = 0;
  if (c->h_fuse_err[0])
    return fail(c, PARD_ERR_DEVICE, "a QKV+attention launch's wait exceeded its spin limit: results are invalid");
  if (c->h_fuse_err[32]) {
    // reported once: the flag is cleared for the calls that follow
    HIP_TRY(c, hipMemsetAsync(c->fuse_err + 32, 0, sizeof(int), c->stream));
    HIP_TRY(c, hipStreamSynchronize(c->stream));
    return fail(c, PARD_ERR_RANGE, "an activation exceeded fp16's range (or was NaN): this call's tokens and the "
                "sequences' caches are invalid; prefill them again");
  }
  return PARD_OK;
}

pard_status pull_seq_sync(pard_ctx* c, int seq) { return pull_seqs_sync(c, &seq, 1); }

// Appends one sequence's rows to a host-built pass: n_ids tokens then n_masks
// mask rows at positions pos0.., the first n_real committed; lm rows are rows
// lm_first .. lm_first + lm_rows - 1 of the sequence.
void append_seq(FwdDesc& d, int slot, const int* ids, int n_ids, int n_masks, int mask_id, int pos0, int n_real,
                int lm_first, int lm_rows) {
  PassSeq& q = d.seq[d.n_seq++];
  q.slot = slot;
  q.row0 = d.n_rows;
  q.n_rows = n_ids + n_masks;
  q.n_real = n_real;
  q.pos0 = pos0;
  q.lm0 = d.n_lm;
  q.lm_rows = lm_rows;
  for (int i = 0; i < q.n_rows; ++i) {
    const int r = q.row0 + i;
    d.ids[r] = i < n_ids ? ids[i] : mask_id;
    d.pos[r] = pos0 + i;
    d.slot[r] = slot;
  }
  for (int j = 0; j < lm_rows; ++j) d.lm_src[q.lm0 + j] = q.row0 + lm_first + j;
  d.n_rows += q.n_rows;
  d.n_lm += lm_rows;
}

FwdDesc make_desc(int slot, const int* ids, int n_ids, int n_masks, int mask_id, int pos0, int n_real, int lm_first,
                  int lm_rows) {
  FwdDesc d{};
  append_seq(d, slot, ids, n_ids, n_masks, mask_id, pos0, n_real, lm_first, lm_rows);
  return d;
}

// Ingest tokens[0..n) at positions pos0.. into model w's cache of one slot (no lm_head).
pard_status ingest(pard_ctx* c, int w, int seq, const int* tokens, int n, int pos0) {
  for (int off = 0; off < n; off += kPrefillRows) {
    const int rows = std::min(kPrefillRows, n - off);
    pard_status st = stage_desc(c, w, make_desc(seq, tokens + off, rows, 0, 0, pos0 + off, rows, rows - 1, 1));
    if (st != PARD_OK) return st;
    PassSpec ps;
    ps.max_rows = rows;
    ps.l_bound = pos0 + off + rows;
    st = forward(c, w, ps);
    if (st != PARD_OK) return st;
  }
  return PARD_OK;
}

bool ids_ok(const int* ids, int n, int vocab) {
  for (int i = 0; i < n; ++i)
    if (ids[i] < 0 || ids[i] >= vocab) return false;
  return true;
}

pard_status check_seq(pard_ctx* c, int seq, bool need_prefill) {
  if (seq < 0 || seq >= c->max_batch) return fail(c, PARD_ERR_CAPACITY, "seq %d outside [0, max_batch=%d)", seq, c->max_batch);
  if (need_prefill && !c->prefilled[seq]) return fail(c, PARD_ERR_STATE, "sequence slot %d is not prefilled", seq);
  return PARD_OK;
}

// Upper bound of the context length used to plan attention for a batch of
// steps (one captured step graph per class): multiples of 1024 keys.
int attn_l_class(int l) {
  return ceil_div(l, 1024) * 1024;
}

// Pass bounds of one fused step over n_seq sequences.
struct StepShape {
  int n_seq = 1, K = 0;
  int draft_rows = 0;     // bound of the (first) draft pass's rows
  int l_class = 0;
  bool vsd = false;       // vanilla speculative decoding: K one-row draft passes
};

// One fused step: draft pass (pending + K-1 masks per sequence) then verify
// pass, each followed by its argmax tail; K = 0 runs the verify pass only.
pard_status step_passes(pard_ctx* c, const StepShape& sh) {
  pard_status st;
  const int K = sh.K, n = sh.n_seq;
  if (K > 0 && sh.vsd) {
    // vanilla drafting (eq. 3): K passes of one row per sequence, the first
    // also ingesting the tokens the draft has not seen
    for (int j = 0; j < K; ++j) {
      PassSpec pd;
      pd.max_rows = j == 0 ? sh.draft_rows : n;
      pd.max_lm_rows = n;
      pd.n_seq = n;
      pd.max_seq_rows = j == 0 ? (n > 1 ? 2 : sh.draft_rows) : 1;
      pd.l_bound = sh.l_class;
      pd.tail = TAIL_VSD_DRAFT;
      pd.next_desc = c->m[j + 1 < K ? PARD_DRAFT : PARD_TARGET].desc;
      if ((st = forward(c, PARD_DRAFT, pd)) != PARD_OK) return st;
    }
  } else if (K > 0) {
    PassSpec pd;
    pd.max_rows = sh.draft_rows;
    pd.typ_rows = n * K;
    pd.max_lm_rows = n * K;
    pd.n_seq = n;
    pd.max_seq_rows = n > 1 ? 2 * K : sh.draft_rows;
    pd.l_bound = sh.l_class;
    pd.tail = TAIL_DRAFT;
    pd.next_desc = c->m[PARD_TARGET].desc;
    if ((st = forward(c, PARD_DRAFT, pd)) != PARD_OK) return st;
  }
  PassSpec pv;
  pv.max_rows = n * (K + 1);
  pv.max_lm_rows = n * (K + 1);
  pv.n_seq = n;
  pv.max_seq_rows = K + 1;
  pv.l_bound = sh.l_class;
  pv.tail = TAIL_VERIFY;
  pv.next_desc = c->m[K > 0 ? PARD_DRAFT : PARD_TARGET].desc;
  pv.emit = true;
  return forward(c, PARD_TARGET, pv);
}

// Replays the captured step for (n_seq, K, l_class), capturing it on first
// use; the sequences themselves come from the device descriptors.  A capture
// failure switches the context to eager launches.
pard_status launch_step_graph(pard_ctx* c, const StepShape& sh) {
  for (const auto& g : c->graphs)
    if (g.n_seq == sh.n_seq && g.k == sh.K && g.l_class == sh.l_class && g.vsd == sh.vsd) {
      HIP_TRY(c, hipGraphLaunch(g.exec, c->stream));
      return PARD_OK;
    }
  if (!c->cap_stream && hipStreamCreateWithFlags(&c->cap_stream, hipStreamNonBlocking) != hipSuccess) {
    c->use_graphs = false;
    return step_passes(c, sh);
  }
  hipStream_t user = c->stream;
  hipGraph_t graph = nullptr;
  hipGraphExec_t exec = nullptr;
  bool ok = hipStreamBeginCapture(c->cap_stream, hipStreamCaptureModeThreadLocal) == hipSuccess;
  if (ok) {
    c->stream = c->cap_stream;
    const pard_status st = step_passes(c, sh);
    c->stream = user;
    ok = hipStreamEndCapture(c->cap_stream, &graph) == hipSuccess && st == PARD_OK && graph;
  }
  ok = ok && hipGraphInstantiate(&exec, graph, nullptr, nullptr, 0) == hipSuccess;
  if (graph) (void)hipGraphDestroy(graph);
  (void)hipGetLastError();
  if (!ok) {
    c->use_graphs = false;
    return step_passes(c, sh);
  }
  c->graphs.push_back({sh.n_seq, sh.K, sh.l_class, sh.vsd, exec});
  HIP_TRY(c, hipGraphLaunch(exec, c->stream));
  return PARD_OK;
}

}  // namespace

// ============================================================================
// C ABI
// ============================================================================

extern "C" {

const char* pard_status_string(pard_status s) {
  switch (s) {
    case PARD_OK: return "PARD_OK";
    case PARD_ERR_ARG: return "PARD_ERR_ARG";
    case PARD_ERR_STATE: return "PARD_ERR_STATE";
    case PARD_ERR_CAPACITY: return "PARD_ERR_CAPACITY";
    case PARD_ERR_NOMEM: return "PARD_ERR_NOMEM";
    case PARD_ERR_DEVICE: return "PARD_ERR_DEVICE";
    case PARD_ERR_UNSUPPORTED: return "PARD_ERR_UNSUPPORTED";
    case PARD_ERR_RANGE: return "PARD_ERR_RANGE";
  }
  return "PARD_UNKNOWN";
}

size_t pard_arena_bytes(const pard_model_spec* target, const pard_model_spec* draft, int32_t max_batch,
                        int32_t max_ctx, int32_t max_k) {
  std::string why;
  const int mask = target ? target->vocab - 1 : 0;
  if (check_all(target, draft, mask, max_batch, max_ctx, max_k, &why) != PARD_OK) return 0;
  pard_ctx tmp;
  tmp.max_batch = max_batch;
  tmp.max_ctx = max_ctx;
  tmp.max_k = max_k;
  tmp.kv_cap = ceil_div(max_ctx, 32) * 32;
  derive(tmp.m[0], *target, max_ctx);
  derive(tmp.m[1], *draft, max_ctx);
  return layout(&tmp, nullptr);
}

pard_status pard_model_load(const pard_model_spec* target, const pard_model_spec* draft, int32_t mask_id,
                            int32_t max_batch, int32_t max_ctx, int32_t max_k, void* dev_arena,
                            size_t arena_bytes, void* hip_stream, pard_ctx** out) {
  if (!out) return PARD_ERR_ARG;
  *out = nullptr;
  std::string why;
  pard_status st = check_all(target, draft, mask_id, max_batch, max_ctx, max_k, &why);
  if (st != PARD_OK) return st;
  if (!dev_arena || (reinterpret_cast<uintptr_t>(dev_arena) & 255)) return PARD_ERR_ARG;
  const size_t need = pard_arena_bytes(target, draft, max_batch, max_ctx, max_k);
  if (arena_bytes < need) return PARD_ERR_NOMEM;

  pard_ctx* c = new (std::nothrow) pard_ctx();
  if (!c) return PARD_ERR_NOMEM;
  c->mask_id = mask_id;
  c->max_batch = max_batch;
  c->max_ctx = max_ctx;
  c->max_k = max_k;
  c->kv_cap = ceil_div(max_ctx, 32) * 32;
  c->stream = reinterpret_cast<hipStream_t>(hip_stream);
  c->arena = static_cast<char*>(dev_arena);
  c->arena_bytes = arena_bytes;
  derive(c->m[0], *target, max_ctx);
  derive(c->m[1], *draft, max_ctx);
  layout(c, c->arena);
  c->hist.assign(max_batch, {});
  if (const char* e = getenv("PARD_NO_GRAPH")) c->use_graphs = e[0] == '0';
  if (const char* e = getenv("PARD_NO_FUSE")) c->use_fused = e[0] == '0';
  if (const char* e = getenv("PARD_NO_FUSE_O")) c->use_fused_o = e[0] == '0';
  if (const char* e = getenv("PARD_NO_FUSE_GU")) c->use_fused_gu = e[0] == '0';
  if (const char* e = getenv("PARD_NO_FUSE_D")) c->use_fused_d = e[0] == '0';
  if (const char* e = getenv("PARD_GU_PRE")) c->gu_pre = atoi(e);
  if (const char* e = getenv("PARD_GU_PRE_Q")) c->gu_pre_q = atoi(e);
  c->prefilled.assign(max_batch, 0);
  c->draft_k.assign(max_batch, 0);

  auto bail = [&](pard_status s) {
    pard_free(c);
    return s;
  };
  if (hipHostMalloc((void**)&c->h_desc, sizeof(FwdDesc) * kDescRing, hipHostMallocDefault) != hipSuccess ||
      hipHostMalloc((void**)&c->h_seq, sizeof(SeqState) * max_batch, hipHostMallocDefault) != hipSuccess ||
      hipHostMalloc((void**)&c->h_gather_idx, sizeof(size_t) * kGatherMax, hipHostMallocDefault) != hipSuccess ||
      hipHostMalloc((void**)&c->h_gather_out, sizeof(float) * kGatherMax, hipHostMallocDefault) != hipSuccess ||
      hipHostMalloc((void**)&c->h_out, sizeof(int) * max_ctx, hipHostMallocDefault) != hipSuccess ||
      hipHostMalloc((void**)&c->h_clock, sizeof(PhaseClock), hipHostMallocDefault) != hipSuccess ||
      hipHostMalloc((void**)&c->h_fuse_err, sizeof(int) * 64, hipHostMallocDefault) != hipSuccess)
    return bail(PARD_ERR_DEVICE);
  {
    int dev = 0, khz = 0;
    if (hipGetDevice(&dev) != hipSuccess || hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, dev) != hipSuccess ||
        khz <= 0)
      return bail(PARD_ERR_DEVICE);
    c->clock_khz = khz;
  }
  memset(c->h_seq, 0, sizeof(SeqState) * max_batch);
  if (hipEventCreate(&c->ev_start) != hipSuccess || hipEventCreate(&c->ev_stop) != hipSuccess)
    return bail(PARD_ERR_DEVICE);

  for (int w = 0; w < 2; ++w)
    if (generate(c, w) != PARD_OK) return bail(PARD_ERR_DEVICE);
  // occupancy of the fused QKV+attention kernels, asked once here rather than
  // during a graph capture
  for (int w = 0; w < 2; ++w)
    for (int mt = 1; mt <= 4; ++mt)
      for (int S = 1; S <= 2; ++S) {
        (void)qkv_attn_capacity(mt, S, c->m[w].spec.head_dim);
        if (mt == 1) {
          const ModelDev& M = c->m[w];
          (void)qkv_attn_capacity(mt, S, M.spec.head_dim, M.p_o.kb_total);
          const int S_gu = pick_S(EPI_SWIGLU, M.p_gu.n_strips, 1);
          for (int d_S = 0; d_S <= 1; ++d_S) {
            const int pre_max = qkv_attn_gu_pre_max(S, M.spec.head_dim, M.p_o.kb_total, S_gu, d_S);
            for (int pre = 1; pre <= pre_max; ++pre)
              (void)qkv_attn_capacity(mt, S, M.spec.head_dim, M.p_o.kb_total, S_gu, pre, d_S);
          }
        }
      }
  if (hipMemsetAsync(c->seq_dev, 0, sizeof(SeqState) * max_batch, c->stream) != hipSuccess ||
      hipMemsetAsync(c->m[0].lm_map, 0, sizeof(int2) * max_batch, c->stream) != hipSuccess ||
      hipMemsetAsync(c->m[1].lm_map, 0, sizeof(int2) * max_batch, c->stream) != hipSuccess ||
      hipMemsetAsync(c->split_counters, 0, sizeof(int) * kSplitCounters, c->stream) != hipSuccess ||
      hipMemsetAsync(c->clock_dev, 0, sizeof(PhaseClock), c->stream) != hipSuccess ||
      hipMemsetAsync(c->fuse_cnt, 0, sizeof(int) * kFuseInts * (c->m[0].spec.n_layers + c->m[1].spec.n_layers),
                     c->stream) != hipSuccess ||
      hipMemsetAsync(c->fuse_err, 0, sizeof(int) * 64, c->stream) != hipSuccess ||
      hipStreamSynchronize(c->stream) != hipSuccess)
    return bail(PARD_ERR_DEVICE);
  *out = c;
  return PARD_OK;
}

void pard_free(pard_ctx* c) {
  if (!c) return;
  (void)hipStreamSynchronize(c->stream);
  if (c->h_desc) (void)hipHostFree(c->h_desc);
  if (c->h_seq) (void)hipHostFree(c->h_seq);
  if (c->h_gather_idx) (void)hipHostFree(c->h_gather_idx);
  if (c->h_gather_out) (void)hipHostFree(c->h_gather_out);
  if (c->h_out) (void)hipHostFree(c->h_out);
  if (c->h_clock) (void)hipHostFree(c->h_clock);
  if (c->h_fuse_err) (void)hipHostFree(c->h_fuse_err);
  if (c->ev_start) (void)hipEventDestroy(c->ev_start);
  if (c->ev_stop) (void)hipEventDestroy(c->ev_stop);
  for (hipEvent_t e : c->timer_ev) (void)hipEventDestroy(e);
  for (auto& g : c->graphs) (void)hipGraphExecDestroy(g.exec);
  if (c->cap_stream) (void)hipStreamDestroy(c->cap_stream);
  delete c;
}

const char* pard_last_error(const pard_ctx* c) { return c ? c->err.c_str() : "null context"; }

pard_status pard_set_sampling(pard_ctx* c, float temperature, uint64_t seed) {
  if (!c) return PARD_ERR_ARG;
  if (!(temperature >= 0.f) || !std::isfinite(temperature) || (temperature > 0.f && temperature < 1e-3f))
    return fail(c, PARD_ERR_ARG, "set_sampling: temperature %g outside {0} and [1e-3, inf)", (double)temperature);
  if (temperature > 0.f && c->m[0].spec.vocab > kMaxSampleVocab)
    return fail(c, PARD_ERR_UNSUPPORTED, "set_sampling: vocab above %d", kMaxSampleVocab);
  c->samp_k = temperature > 0.f ? (float)(1.4426950408889634 / temperature) : 0.f;
  c->samp_seed = seed;
  // captured steps hold the old settings in their kernel arguments
  if (hipStreamSynchronize(c->stream) != hipSuccess) return fail(c, PARD_ERR_DEVICE, "set_sampling: stream");
  for (auto& g : c->graphs) (void)hipGraphExecDestroy(g.exec);
  c->graphs.clear();
  return PARD_OK;
}

pard_status pard_prefill(pard_ctx* c, int32_t seq, const int32_t* prompt, int32_t n, int32_t* first_token) {
  if (!c) return PARD_ERR_ARG;
  pard_status st = check_seq(c, seq, false);
  if (st != PARD_OK) return st;
  if (!prompt || !first_token || n < 1) return fail(c, PARD_ERR_ARG, "prefill: null pointer or empty prompt");
  if (!ids_ok(prompt, n, c->m[0].spec.vocab)) return fail(c, PARD_ERR_ARG, "prefill: token id out of range");
  if ((int64_t)n + 2 * c->max_k + 1 > c->max_ctx)
    return fail(c, PARD_ERR_CAPACITY, "prefill: prompt of %d does not fit max_ctx=%d", n, c->max_ctx);
  SeqState& S = c->h_seq[seq];
  memset(&S, 0, sizeof S);
  S.L[0] = n;
  S.L[1] = n;
  S.mask_id = c->mask_id;
  if ((st = push_seq(c, seq)) != PARD_OK) return st;
  for (int w = 1; w >= 0; --w) {   // draft first, the target's last chunk sets the first token
    for (int off = 0; off < n; off += kPrefillRows) {
      const int rows = std::min(kPrefillRows, n - off);
      const bool last = (off + rows == n) && w == PARD_TARGET;
      st = stage_desc(c, w, make_desc(seq, prompt + off, rows, 0, 0, off, rows, rows - 1, 1));
      if (st != PARD_OK) return st;
      PassSpec ps;
      ps.max_rows = rows;
      ps.l_bound = off + rows;
      if (last) {
        ps.max_lm_rows = 1;
        ps.tail = TAIL_PREFILL;
      }
      if ((st = forward(c, w, ps)) != PARD_OK) return st;
    }
  }
  if ((st = pull_seq_sync(c, seq)) != PARD_OK) return st;
  *first_token = S.bonus;
  c->hist[seq].assign(prompt, prompt + n);
  c->hist[seq].push_back(S.bonus);
  c->prefilled[seq] = 1;
  c->draft_k[seq] = 0;
  return PARD_OK;
}

pard_status pard_draft(pard_ctx* c, int32_t seq, const int32_t* prefix, int32_t n_prefix, int32_t K,
                       int32_t* cand) {
  if (!c) return PARD_ERR_ARG;
  pard_status st = check_seq(c, seq, true);
  if (st != PARD_OK) return st;
  if (!prefix || !cand || n_prefix < 1) return fail(c, PARD_ERR_ARG, "draft: null pointer or empty prefix");
  if (K < 1 || K > c->max_k) return fail(c, PARD_ERR_ARG, "draft: K=%d outside [1, max_k=%d]", K, c->max_k);
  if (!ids_ok(prefix, n_prefix, c->m[1].spec.vocab)) return fail(c, PARD_ERR_ARG, "draft: token id out of range");
  if ((int64_t)n_prefix + K - 1 > c->max_ctx)
    return fail(c, PARD_ERR_CAPACITY, "draft: %d rows past position %d exceed max_ctx", K - 1, n_prefix);
  SeqState& S = c->h_seq[seq];
  const SeqState saved = S;
  int Ld = std::min(S.L[1], n_prefix - 1);
  // a long unseen tail is ingested first so that the draft pass fits kMaxRows rows
  const int max_real = kMaxRows - (K - 1);
  if (n_prefix - Ld > max_real) {
    const int extra = n_prefix - Ld - max_real;
    if ((st = ingest(c, PARD_DRAFT, seq, prefix + Ld, extra, Ld)) != PARD_OK) { S = saved; return st; }
    Ld += extra;
  }
  const int n_new = n_prefix - Ld;
  S.k = K;
  S.vsd = 0;
  S.L[1] = Ld;
  if ((st = push_seq(c, seq)) != PARD_OK) { S = saved; return st; }
  const FwdDesc d = make_desc(seq, prefix + Ld, n_new, K - 1, c->mask_id, Ld, n_new, n_new - 1, K);
  if ((st = stage_desc(c, PARD_DRAFT, d)) != PARD_OK) { S = saved; return st; }
  PassSpec ps;
  ps.max_rows = d.n_rows;
  ps.l_bound = Ld + d.n_rows;
  ps.max_lm_rows = K;
  ps.tail = TAIL_DRAFT;
  ps.next_desc = c->m[PARD_TARGET].desc;
  if ((st = forward(c, PARD_DRAFT, ps)) != PARD_OK) { S = saved; return st; }
  if ((st = pull_seq_sync(c, seq)) != PARD_OK) return st;
  for (int i = 0; i < K; ++i) cand[i] = S.cand[i];
  c->draft_k[seq] = K;
  return PARD_OK;
}

pard_status pard_verify(pard_ctx* c, int32_t seq, const int32_t* cand, int32_t K, int32_t* n_accepted,
                        int32_t* bonus) {
  if (!c) return PARD_ERR_ARG;
  pard_status st = check_seq(c, seq, true);
  if (st != PARD_OK) return st;
  if (!n_accepted || !bonus || (K > 0 && !cand)) return fail(c, PARD_ERR_ARG, "verify: null pointer");
  if (K < 0 || K > c->max_k) return fail(c, PARD_ERR_ARG, "verify: K=%d outside [0, max_k=%d]", K, c->max_k);
  if (K > 0 && !ids_ok(cand, K, c->m[0].spec.vocab)) return fail(c, PARD_ERR_ARG, "verify: token id out of range");
  SeqState& S = c->h_seq[seq];
  if ((int64_t)S.L[0] + K + 1 > c->max_ctx)
    return fail(c, PARD_ERR_CAPACITY, "verify: %d rows at position %d exceed max_ctx", K + 1, S.L[0]);
  if (c->samp_k > 0.f && K > 0 && c->draft_k[seq] != K)
    return fail(c, PARD_ERR_STATE, "verify: sampling needs this slot's draft pass of the same K=%d first", K);
  const SeqState saved = S;
  const int Lt = S.L[0];
  int ids[kMaxK + 1];
  ids[0] = S.bonus;
  for (int i = 0; i < K; ++i) {
    ids[1 + i] = cand[i];
    S.cand[i] = cand[i];
  }
  S.k = K;
  S.vsd = 0;
  if ((st = push_seq(c, seq)) != PARD_OK) { S = saved; return st; }
  if ((st = stage_desc(c, PARD_TARGET, make_desc(seq, ids, K + 1, 0, 0, Lt, K + 1, 0, K + 1))) != PARD_OK) {
    S = saved;
    return st;
  }
  PassSpec ps;
  ps.max_rows = K + 1;
  ps.l_bound = Lt + K + 1;
  ps.max_lm_rows = K + 1;
  ps.tail = TAIL_VERIFY;
  ps.next_desc = c->m[K > 0 ? PARD_DRAFT : PARD_TARGET].desc;
  if ((st = forward(c, PARD_TARGET, ps)) != PARD_OK) { S = saved; return st; }
  if ((st = pull_seq_sync(c, seq)) != PARD_OK) return st;
  *n_accepted = S.a;
  *bonus = S.bonus;
  c->draft_k[seq] = 0;
  std::vector<int>& h = c->hist[seq];
  h.resize(Lt + 1);
  for (int i = 0; i < S.a; ++i) h.push_back(cand[i]);
  h.push_back(S.bonus);
  return PARD_OK;
}

pard_status pard_kv_truncate(pard_ctx* c, int32_t seq, int32_t which, int32_t new_len) {
  if (!c) return PARD_ERR_ARG;
  pard_status st = check_seq(c, seq, true);
  if (st != PARD_OK) return st;
  if (which != PARD_TARGET && which != PARD_DRAFT) return fail(c, PARD_ERR_ARG, "truncate: bad model id");
  SeqState& S = c->h_seq[seq];
  if (new_len < 0 || new_len > S.L[which])
    return fail(c, PARD_ERR_ARG, "truncate: new_len %d outside [0, %d]", new_len, S.L[which]);
  const SeqState saved = S;
  S.L[which] = new_len;
  if ((st = push_seq(c, seq)) != PARD_OK || (st = pull_seq_sync(c, seq)) != PARD_OK) {
    S = saved;
    return st;
  }
  if (which == PARD_TARGET) {
    std::vector<int>& h = c->hist[seq];
    const int pending = h.back();
    h.resize(new_len);
    h.push_back(pending);
  }
  return PARD_OK;
}

pard_status pard_kv_len(const pard_ctx* c, int32_t seq, int32_t which, int32_t* len) {
  if (!c || !len || (which != PARD_TARGET && which != PARD_DRAFT)) return PARD_ERR_ARG;
  if (seq < 0 || seq >= c->max_batch) return PARD_ERR_CAPACITY;
  *len = c->h_seq[seq].L[which];
  return PARD_OK;
}

pard_status pard_generate(pard_ctx* c, int32_t n_seq, const int32_t* seqs, int32_t K, int32_t n_tokens,
                          int32_t max_steps, int32_t* out_tokens, pard_stats* stats) {
  return pard_generate_ex(c, n_seq, seqs, K, PARD_MODE_PARALLEL, n_tokens, max_steps, out_tokens, stats);
}

pard_status pard_generate_ex(pard_ctx* c, int32_t n_seq, const int32_t* seqs, int32_t K, int32_t mode,
                             int32_t n_tokens, int32_t max_steps, int32_t* out_tokens, pard_stats* stats) {
  if (!c) return PARD_ERR_ARG;
  if (mode != PARD_MODE_PARALLEL && mode != PARD_MODE_VANILLA) return fail(c, PARD_ERR_ARG, "generate: bad mode %d", mode);
  const bool vsd = mode == PARD_MODE_VANILLA;
  if (vsd && c->samp_k > 0.f)
    return fail(c, PARD_ERR_UNSUPPORTED, "generate: vanilla drafting runs greedy only (sampling is set)");
  if (!seqs || !out_tokens || n_tokens < 1) return fail(c, PARD_ERR_ARG, "generate: null pointer or n_tokens < 1");
  if (n_seq < 1 || n_seq > std::min(c->max_batch, kMaxPassSeqs))
    return fail(c, PARD_ERR_CAPACITY, "generate: n_seq=%d outside [1, %d]", n_seq, std::min(c->max_batch, kMaxPassSeqs));
  if (K < 0 || K > c->max_k) return fail(c, PARD_ERR_ARG, "generate: K=%d outside [0, max_k=%d]", K, c->max_k);
  if (n_seq > 1 && (n_seq * 2 * K > kMaxPassRows || n_seq * (K + 1) > c->lm_rows_cap))
    return fail(c, PARD_ERR_CAPACITY, "generate: %d sequences at K=%d exceed %d rows per pass", n_seq, K,
                kMaxPassRows);
  pard_status st;
  for (int i = 0; i < n_seq; ++i) {
    if ((st = check_seq(c, seqs[i], true)) != PARD_OK) return st;
    for (int j = 0; j < i; ++j)
      if (seqs[j] == seqs[i]) return fail(c, PARD_ERR_ARG, "generate: slot %d listed twice", seqs[i]);
    const int Lt = c->h_seq[seqs[i]].L[0];
    if ((int64_t)Lt + n_tokens + 2 * K + 1 > c->max_ctx)
      return fail(c, PARD_ERR_CAPACITY, "generate: %d tokens from length %d may exceed max_ctx=%d", n_tokens, Lt,
                  c->max_ctx);
  }
  std::vector<SeqState> saved(n_seq);
  for (int i = 0; i < n_seq; ++i) saved[i] = c->h_seq[seqs[i]];
  auto restore = [&](pard_status s) {
    for (int i = 0; i < n_seq; ++i) c->h_seq[seqs[i]] = saved[i];
    return s;
  };
  // every draft catches up with the committed tokens it has not seen; a
  // sequence's first draft pass holds at most kMaxRows rows alone, 2K in a batch
  FwdDesc first{};
  for (int i = 0; i < n_seq; ++i) {
    const int seq = seqs[i];
    SeqState& S = c->h_seq[seq];
    const std::vector<int>& hist = c->hist[seq];
    const int Lt = S.L[0];
    int Ld = std::min(S.L[1], Lt);
    if (K > 0) {
      const int total = Lt + 1;                  // committed tokens + pending
      // pending rows of the first draft pass: PARD adds K-1 mask rows, a
      // vanilla pass none (later vanilla passes see at most 2 pending tokens)
      const int max_first = vsd ? (n_seq == 1 ? kMaxRows : 2) : (n_seq == 1 ? kMaxRows : 2 * K) - (K - 1);
      if (total - Ld > max_first) {
        const int extra = total - Ld - max_first;
        if ((st = ingest(c, PARD_DRAFT, seq, hist.data() + Ld, extra, Ld)) != PARD_OK) return restore(st);
        Ld += extra;
      }
      S.n_pending = total - Ld;
      for (int j = 0; j < S.n_pending; ++j) S.pending[j] = hist[Ld + j];
    }
    S.L[1] = Ld;
    S.k = K;
    S.vsd = vsd && K > 0 ? 1 : 0;
    S.j = 0;
    S.n_out = 1;
    S.n_target = n_tokens;
    S.steps = 0;
    S.mask_id = c->mask_id;
    c->draft_k[seq] = 0;
    memset(S.accept_hist, 0, sizeof S.accept_hist);
    if ((st = push_seq(c, seq)) != PARD_OK) return restore(st);
    if (K > 0 && vsd) {
      append_seq(first, seq, S.pending, S.n_pending, 0, 0, Ld, S.n_pending, S.n_pending - 1, 1);
    } else if (K > 0) {
      append_seq(first, seq, S.pending, S.n_pending, K - 1, c->mask_id, Ld, S.n_pending, S.n_pending - 1, K);
    } else {
      const int b = S.bonus;
      append_seq(first, seq, &b, 1, 0, 0, Lt, 1, 0, 1);
    }
  }
  if ((st = stage_desc(c, K > 0 ? PARD_DRAFT : PARD_TARGET, first)) != PARD_OK) return restore(st);
  HIP_TRY(c, hipMemsetAsync(c->clock_dev, 0, sizeof(PhaseClock), c->stream));
  HIP_TRY(c, hipEventRecord(c->ev_start, c->stream));
  // active: sequences that still need tokens (a finished one leaves the
  // batch when the device stages the next draft pass)
  std::vector<int> active(seqs, seqs + n_seq);
  int steps = 0;
  bool first_step = true;
  while (!active.empty() && (max_steps <= 0 || steps < max_steps)) {
    int min_left = INT32_MAX, max_L = 0;
    for (int seq : active) {
      min_left = std::min(min_left, n_tokens - c->h_seq[seq].n_out);
      max_L = std::max(max_L, c->h_seq[seq].L[0]);
    }
    int batch = ceil_div(min_left, K + 1);
    if (max_steps > 0) batch = std::min(batch, max_steps - steps);
    // a bounded batch keeps the attention length class (and so the attention
    // plan of the captured steps) close to the actual context
    batch = std::min(batch, kStepsPerPlan);
    // L_t grows by at most K+1 per step: one attention plan covers the batch
    StepShape sh;
    sh.n_seq = (int)active.size();
    sh.K = K;
    sh.vsd = vsd;
    sh.l_class = attn_l_class(max_L + batch * (K + 1) + K + 1);
    for (int i = 0; i < batch; ++i) {
      // a single sequence's first draft pass may carry more pending rows
      if (vsd)
        sh.draft_rows = sh.n_seq > 1 ? sh.n_seq * 2 : (first_step ? std::max(first.n_rows, 2) : 2);
      else
        sh.draft_rows = sh.n_seq > 1 ? sh.n_seq * 2 * K : (first_step ? std::max(first.n_rows, 2 * K) : 2 * K);
      if (first_step || !c->use_graphs || c->timer_class >= 0) {
        if ((st = step_passes(c, sh)) != PARD_OK) return st;
      } else {
        if ((st = launch_step_graph(c, sh)) != PARD_OK) return st;
      }
      first_step = false;
    }
    HIP_TRY(c, hipEventRecord(c->ev_stop, c->stream));
    if ((st = pull_seqs_sync(c, active.data(), (int)active.size())) != PARD_OK) return st;
    std::vector<int> still;
    for (int seq : active) {
      steps = std::max(steps, c->h_seq[seq].steps);
      if (c->h_seq[seq].n_out < n_tokens) still.push_back(seq);
    }
    if (n_seq > 1) active.swap(still);          // batched passes drop finished sequences
    else if (still.empty()) active.clear();
  }
  float ms = 0.f;
  if (steps > 0) HIP_TRY(c, hipEventElapsedTime(&ms, c->ev_start, c->ev_stop));
  HIP_TRY(c, hipMemcpyAsync(c->h_clock, c->clock_dev, sizeof(PhaseClock), hipMemcpyDeviceToHost, c->stream));
  HIP_TRY(c, hipStreamSynchronize(c->stream));
  int64_t total_written = 0;
  int64_t hist_sum[kMaxK + 1] = {0};
  for (int i = 0; i < n_seq; ++i) {
    const int seq = seqs[i];
    SeqState& S = c->h_seq[seq];
    std::vector<int>& hist = c->hist[seq];
    const int produced = S.n_out;
    const int n_new = produced - 1;   // tokens appended after the pending one
    if (n_new > 0) {
      HIP_TRY(c, hipMemcpyAsync(c->h_out, c->out_dev + (size_t)seq * c->max_ctx + 1, sizeof(int) * n_new,
                                hipMemcpyDeviceToHost, c->stream));
      HIP_TRY(c, hipStreamSynchronize(c->stream));
    }
    const int written = std::min(produced, n_tokens);
    int32_t* out = out_tokens + (size_t)i * n_tokens;
    out[0] = hist.back();
    for (int j = 1; j < written; ++j) out[j] = c->h_out[j - 1];
    for (int j = 0; j < n_new; ++j) hist.push_back(c->h_out[j]);
    total_written += written;
    for (int j = 0; j <= kMaxK; ++j) hist_sum[j] += S.accept_hist[j];
  }
  if (stats) {
    memset(stats, 0, sizeof *stats);
    stats->steps = steps;
    stats->tokens = total_written;
    stats->elapsed_ms = ms;
    const PhaseClock& ck = *c->h_clock;
    const double per_ms = c->clock_khz;   // clock ticks per millisecond
    stats->draft_ms = ck.draft_ticks / per_ms;
    stats->verify_ms = ck.verify_ticks / per_ms;
    stats->accept_ms = ck.accept_ticks / per_ms;
    // step latencies: gaps between consecutive verify-tail ends in the ring
    const uint64_t n_end = std::min<uint64_t>(ck.n_steps, kStepRing);
    std::vector<double> lat;
    for (uint64_t i = 1; i < n_end; ++i) {
      const uint64_t j = ck.n_steps - n_end + i;
      lat.push_back((ck.step_end[j % kStepRing] - ck.step_end[(j - 1) % kStepRing]) / per_ms);
    }
    if (!lat.empty()) {
      std::sort(lat.begin(), lat.end());
      auto rank = [&](double q) { return lat[(size_t)std::max(0.0, std::ceil(q * lat.size()) - 1)]; };
      stats->step_ms_p50 = rank(0.5);
      stats->step_ms_p90 = rank(0.9);
    }
    for (int i = 0; i <= kMaxK; ++i) stats->accept_hist[i] = hist_sum[i];
  }
  return PARD_OK;
}

// ----------------------------------------------------------------------------
// COD training-data processing
// ----------------------------------------------------------------------------

namespace {

bool cod_params_ok(int32_t K, double r, double r_min) {
  return K >= 1 && K <= 64 && r > 0.0 && r <= 1.0 && r_min >= 0.0 && r_min <= 1.0 && std::isfinite(r) &&
         std::isfinite(r_min);
}

// Packed rows a sample of n_tokens tokens can produce: n columns of subtask 1
// plus each later subtask's keep target (the same float64 arithmetic as the kernel).
int64_t cod_capacity(int64_t n_tokens, int32_t K, double r, double r_min) {
  const int64_t n = n_tokens - 1;
  int64_t total = n;
  double gamma = 1.0;
  for (int k = 2; k <= K; ++k) {
    gamma *= r;
    total += (int64_t)std::floor((double)n * std::fmax(gamma, r_min) + 0.5);
  }
  return total;
}

}  // namespace

int64_t pard_cod_capacity(int32_t n_tokens, int32_t K, double r, double r_min) {
  if (n_tokens < 2 || n_tokens - 1 > cod_max_columns() || !cod_params_ok(K, r, r_min)) return -1;
  return cod_capacity(n_tokens, K, r, r_min);
}

int64_t pard_cod_layout(const int64_t* tok_offsets, int32_t n_samples, int32_t K, double r, double r_min,
                        int64_t* out_offsets) {
  if (!tok_offsets || !out_offsets || n_samples < 1 || !cod_params_ok(K, r, r_min) || tok_offsets[0] < 0) return -1;
  out_offsets[0] = 0;
  for (int s = 0; s < n_samples; ++s) {
    const int64_t len = tok_offsets[s + 1] - tok_offsets[s];
    if (len < 2 || len - 1 > cod_max_columns()) return -1;
    out_offsets[s + 1] = out_offsets[s] + cod_capacity(len, K, r, r_min);
  }
  return out_offsets[n_samples];
}

size_t pard_cod_workspace_bytes(int32_t n_samples) {
  return n_samples < 1 ? 0 : align256(2 * sizeof(int64_t) * ((size_t)n_samples + 1));
}

}  // extern "C"

namespace {

// Host-side checks of a COD batch (no device work): every sample's length fits
// the kernel and its output region holds its capacity.  *max_cols receives the
// longest sample's column count.
pard_status cod_check(const int32_t* tokens, const int64_t* tok_offsets, int32_t n_samples, int32_t K, double r,
                      double r_min, const int64_t* out_offsets, int32_t* const* outs, int32_t* out_len,
                      int* max_cols) {
  if (!tokens || !tok_offsets || !out_offsets || !out_len || n_samples < 1 || !cod_params_ok(K, r, r_min))
    return PARD_ERR_ARG;
  for (int i = 0; i < 5; ++i)
    if (!outs[i]) return PARD_ERR_ARG;
  if (tok_offsets[0] < 0 || out_offsets[0] < 0) return PARD_ERR_ARG;
  *max_cols = 1;
  for (int s = 0; s < n_samples; ++s) {
    const int64_t len = tok_offsets[s + 1] - tok_offsets[s];
    if (len < 2 || len - 1 > cod_max_columns()) return PARD_ERR_ARG;
    if (out_offsets[s + 1] - out_offsets[s] < cod_capacity(len, K, r, r_min)) return PARD_ERR_CAPACITY;
    *max_cols = std::max(*max_cols, (int)(len - 1));
  }
  return PARD_OK;
}

// Copies both offset arrays to d_off (2 * (n_samples + 1) int64 of device
// memory), runs the kernel on st and waits for it.
pard_status cod_run(const int32_t* tokens, const int64_t* tok_offsets, int32_t n_samples, int32_t K, double r,
                    double r_min, int32_t mask_id, uint64_t seed, const int64_t* out_offsets, int32_t* const* outs,
                    int32_t* out_len, int max_cols, int64_t* d_off, float* kernel_ms, hipStream_t st) {
  const size_t bytes = sizeof(int64_t) * (size_t)(n_samples + 1);
  CodArgs a;
  a.k_max = K;
  a.r = r;
  a.r_min = r_min;
  a.mask_id = mask_id;
  a.seed = seed;
  a.ids = outs[0];
  a.labels = outs[1];
  a.pos = outs[2];
  a.section = outs[3];
  a.column = outs[4];
  a.out_len = out_len;
  pard_status stt = PARD_OK;
  hipEvent_t ev[2] = {nullptr, nullptr};
  if (kernel_ms && (hipEventCreate(&ev[0]) != hipSuccess || hipEventCreate(&ev[1]) != hipSuccess)) stt = PARD_ERR_DEVICE;
  if (stt == PARD_OK &&
      (hipMemcpyAsync(d_off, tok_offsets, bytes, hipMemcpyHostToDevice, st) != hipSuccess ||
       hipMemcpyAsync(d_off + n_samples + 1, out_offsets, bytes, hipMemcpyHostToDevice, st) != hipSuccess ||
       (kernel_ms && hipEventRecord(ev[0], st) != hipSuccess) ||
       launch_cod(tokens, d_off, d_off + n_samples + 1, n_samples, max_cols, a, st) != hipSuccess ||
       (kernel_ms && hipEventRecord(ev[1], st) != hipSuccess) || hipStreamSynchronize(st) != hipSuccess))
    stt = PARD_ERR_DEVICE;
  if (stt == PARD_OK && kernel_ms && hipEventElapsedTime(kernel_ms, ev[0], ev[1]) != hipSuccess) stt = PARD_ERR_DEVICE;
  for (hipEvent_t e : ev)
    if (e) (void)hipEventDestroy(e);
  return stt;
}

// Device scratch of pard_cod_build_noalloc: the device copy of its two offset
// arrays, (n_samples + 1) int64 each, for at most PARD_COD_NOALLOC_MAX_SAMPLES
// samples (1 MiB; every GPU the library runs on holds one until the process
// ends).  Host code never passes `scratch` itself to the device: its name is a
// host-side stand-in, and each GPU's copy has its own device address, looked
// up once per device and kept in g_scratch_dev.
static __device__ __align__(256) int64_t scratch[2 * (PARD_COD_NOALLOC_MAX_SAMPLES + 1)];
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
int64_t* g_scratch_dev[kMaxDevices];

// Device address of the current device's scratch, looked up on the first call
// on that device (with it current) and kept.
pard_status scratch_address(int64_t** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return PARD_ERR_DEVICE;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_dev[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return PARD_ERR_DEVICE;
    g_scratch_dev[dev] = static_cast<int64_t*>(p);
  }
  *out = g_scratch_dev[dev];
  return PARD_OK;
}

}  // namespace

extern "C" {

pard_status pard_cod_build(const int32_t* tokens, const int64_t* tok_offsets, int32_t n_samples, int32_t K, double r,
                           double r_min, int32_t mask_id, uint64_t seed, const int64_t* out_offsets, int32_t* out_ids,
                           int32_t* out_labels, int32_t* out_pos, int32_t* out_section, int32_t* out_column,
                           int32_t* out_len, void* workspace, size_t workspace_bytes, float* kernel_ms,
                           void* hip_stream) {
  int32_t* const outs[5] = {out_ids, out_labels, out_pos, out_section, out_column};
  int max_cols = 1;
  if (!workspace || (reinterpret_cast<uintptr_t>(workspace) & 255) || n_samples < 1) return PARD_ERR_ARG;
  if (workspace_bytes < pard_cod_workspace_bytes(n_samples)) return PARD_ERR_NOMEM;
  const pard_status st = cod_check(tokens, tok_offsets, n_samples, K, r, r_min, out_offsets, outs, out_len, &max_cols);
  if (st != PARD_OK) return st;
  return cod_run(tokens, tok_offsets, n_samples, K, r, r_min, mask_id, seed, out_offsets, outs, out_len, max_cols,
                 static_cast<int64_t*>(workspace), kernel_ms, reinterpret_cast<hipStream_t>(hip_stream));
}

pard_status pard_cod_build_noalloc(const int32_t* tokens, const int64_t* tok_offsets, int32_t n_samples, int32_t K,
                                   double r, double r_min, int32_t mask_id, uint64_t seed, const int64_t* out_offsets,
                                   int32_t* out_ids, int32_t* out_labels, int32_t* out_pos, int32_t* out_section,
                                   int32_t* out_column, int32_t* out_len, void* hip_stream) {
  int32_t* const outs[5] = {out_ids, out_labels, out_pos, out_section, out_column};
  int max_cols = 1;
  if (n_samples > PARD_COD_NOALLOC_MAX_SAMPLES) return PARD_ERR_CAPACITY;
  const pard_status st = cod_check(tokens, tok_offsets, n_samples, K, r, r_min, out_offsets, outs, out_len, &max_cols);
  if (st != PARD_OK) return st;
  int64_t* d_off = nullptr;
  if (scratch_address(&d_off) != PARD_OK) return PARD_ERR_DEVICE;
  return cod_run(tokens, tok_offsets, n_samples, K, r, r_min, mask_id, seed, out_offsets, outs, out_len, max_cols, d_off,
                 nullptr, reinterpret_cast<hipStream_t>(hip_stream));
}

pard_status pard_read_logits(const pard_ctx* cc, int32_t which, int32_t seq, float* out, int32_t rows,
                             int32_t vocab) {
  pard_ctx* c = const_cast<pard_ctx*>(cc);
  if (!c || !out || (which != PARD_TARGET && which != PARD_DRAFT)) return PARD_ERR_ARG;
  if (seq < 0 || seq >= c->max_batch) return fail(c, PARD_ERR_ARG, "read_logits: bad seq");
  const ModelDev& M = c->m[which];
  if (vocab != M.spec.vocab) return fail(c, PARD_ERR_ARG, "read_logits: vocab mismatch");
  int2 lm{0, 0};
  HIP_TRY(c, hipMemcpyAsync(&lm, M.lm_map + seq, sizeof lm, hipMemcpyDeviceToHost, c->stream));
  HIP_TRY(c, hipStreamSynchronize(c->stream));
  if (lm.y == 0) return fail(c, PARD_ERR_STATE, "read_logits: no lm_head pass of this model for slot %d yet", seq);
  if (rows < 1 || rows > lm.y) return fail(c, PARD_ERR_ARG, "read_logits: rows %d outside [1, %d]", rows, lm.y);
  HIP_TRY(c, hipMemcpyAsync(out, M.logits + (size_t)lm.x * vocab, sizeof(float) * rows * vocab, hipMemcpyDeviceToHost,
                            c->stream));
  HIP_TRY(c, hipStreamSynchronize(c->stream));
  return PARD_OK;
}

pard_status pard_read_weight(const pard_ctx* cc, int32_t which, int32_t tensor, int32_t row, int32_t col0,
                             int32_t n, float* out) {
  pard_ctx* c = const_cast<pard_ctx*>(cc);
  if (!c || !out || (which != PARD_TARGET && which != PARD_DRAFT)) return PARD_ERR_ARG;
  if (n < 1 || n > kGatherMax || row < 0 || col0 < 0) return fail(c, PARD_ERR_ARG, "read_weight: bad range");
  const ModelDev& M = c->m[which];
  const pard_model_spec& s = M.spec;
  const int hd = s.head_dim;
  const uint16_t* buf = nullptr;
  int prow = 0, rows = 0, cols = 0, npad = 0;   // npad: packed rows of the buffer
  const float* fbuf = nullptr;
  auto qk_row = [&](int r) { const int head = r / hd, dim = r % hd; return head * hd + (dim < hd / 2 ? 2 * dim : 2 * (dim - hd / 2) + 1); };
  if (tensor == 0 || (tensor == 1 && !s.tied_embeddings)) {
    buf = tensor == 0 ? M.embed : M.lm_head;
    rows = s.vocab; cols = M.d; npad = s.vocab; prow = row;
  } else if (tensor >= 16 && tensor / 16 - 1 < s.n_layers) {
    const int l = tensor / 16 - 1, j = tensor % 16;
    const Layer& L = M.layers[l];
    switch (j) {
      case 0: buf = L.wqkv; rows = M.q_dim; cols = M.d; npad = M.nqkv; prow = qk_row(row); break;
      case 1: buf = L.wqkv; rows = M.kv_dim; cols = M.d; npad = M.nqkv; prow = M.q_dim + qk_row(row); break;
      case 2: buf = L.wqkv; rows = M.kv_dim; cols = M.d; npad = M.nqkv; prow = M.q_dim + M.kv_dim + row; break;
      case 3: buf = L.wo; rows = M.d; cols = M.q_dim; npad = M.d; prow = row; break;
      case 4: buf = L.wgu; rows = s.ffn_dim; cols = M.d; npad = 2 * M.f_pad; prow = (row / 8) * 16 + row % 8; break;
      case 5: buf = L.wgu; rows = s.ffn_dim; cols = M.d; npad = 2 * M.f_pad; prow = (row / 8) * 16 + 8 + row % 8; break;
      case 6: buf = L.wd; rows = M.d; cols = s.ffn_dim; npad = M.d; prow = row; break;
      case 7: case 8: case 9:
        if (!L.bqkv) return fail(c, PARD_ERR_ARG, "read_weight: model has no bias");
        fbuf = L.bqkv; cols = 1;
        rows = j == 7 ? M.q_dim : M.kv_dim;
        prow = j == 7 ? qk_row(row) : (j == 8 ? M.q_dim + qk_row(row) : M.q_dim + M.kv_dim + row);
        break;
      default: return fail(c, PARD_ERR_ARG, "read_weight: bad tensor ordinal");
    }
  } else {
    return fail(c, PARD_ERR_ARG, "read_weight: bad tensor ordinal");
  }
  if (row >= rows || col0 + n > cols) return fail(c, PARD_ERR_ARG, "read_weight: range outside the tensor");
  if (fbuf) {
    HIP_TRY(c, hipMemcpy(out, fbuf + prow, sizeof(float), hipMemcpyDeviceToHost));
    return PARD_OK;
  }
  const size_t n_strips = (size_t)npad / 16;
  for (int i = 0; i < n; ++i) {
    const int col = col0 + i;
    const size_t strip = prow / 16, kb = col / 32;
    const int lane = (prow % 16) + 16 * ((col % 32) / 8);
    c->h_gather_idx[i] = ((kb * n_strips + strip) * 64 + lane) * 8 + (col % 8);
  }
  HIP_TRY(c, hipMemcpyAsync(c->gather_idx_dev, c->h_gather_idx, sizeof(size_t) * n, hipMemcpyHostToDevice, c->stream));
  HIP_TRY(c, launch_gather_u16(buf, c->gather_idx_dev, n, c->gather_out_dev, c->stream));
  HIP_TRY(c, hipMemcpyAsync(out, c->gather_out_dev, sizeof(float) * n, hipMemcpyDeviceToHost, c->stream));
  HIP_TRY(c, hipStreamSynchronize(c->stream));
  return PARD_OK;
}

pard_status pard_timer_enable(pard_ctx* c, int32_t kernel_class, int32_t max_launches) {
  if (!c) return PARD_ERR_ARG;
  HIP_TRY(c, hipStreamSynchronize(c->stream));
  c->timer_class = -1;
  c->timer_used = 0;
  c->timer_max = 0;
  if (kernel_class < 0) return PARD_OK;
  if (kernel_class >= 16 || max_launches < 1 || max_launches > 1 << 16)
    return fail(c, PARD_ERR_ARG, "timer: bad class or launch count");
  while ((int)c->timer_ev.size() < 2 * max_launches) {
    hipEvent_t e;
    HIP_TRY(c, hipEventCreate(&e));
    c->timer_ev.push_back(e);
  }
  c->timer_class = kernel_class;
  c->timer_max = max_launches;
  return PARD_OK;
}

pard_status pard_timer_read(pard_ctx* c, int32_t* launches, double* total_ms) {
  if (!c || !launches || !total_ms) return PARD_ERR_ARG;
  HIP_TRY(c, hipStreamSynchronize(c->stream));
  double sum = 0;
  for (int i = 0; i < c->timer_used; ++i) {
    float ms = 0;
    HIP_TRY(c, hipEventElapsedTime(&ms, c->timer_ev[2 * i], c->timer_ev[2 * i + 1]));
    sum += ms;
  }
  *launches = c->timer_used;
  *total_ms = sum;
  return PARD_OK;
}

}  // extern "C"
