// Stand-alone launches of the one-launch decode layer (k_qkv_attn: QKV GEMM,
// attention, O-projection, gate/up and down GEMMs), for hardware counters
// and launch timing.
//
// Builds one layer's operands at the 8B-target or 1B-draft shape of the
// benchmark pair (LLaMA3.1-8B: d 4096, 32 query / 8 KV heads of 128, FFN
// 14336; LLaMA3.2-1B: d 2048, 32 / 8 heads of 64, FFN 8192), with the tile
// plan the engine uses for a decode pass of that shape (8B: the verify pass,
// 9 rows; 1B: the draft pass, 8 rows planned as 16), its rows at positions
// context.. (default 1142, the mean committed length of the benchmark's
// timed decode steps), and launches it through launch_qkv_attn 20 times untimed
// and 100 times timed (each launch alone, between HIP events, after its
// counters are zeroed).  `copies` > 1 cycles the launches through that many
// copies of the layer's weights, so that they are not served from the caches
// as they would not be in a decode step.  Weights and activations are seeded
// pseudo-random fp16 values: the numerics of the launch are tested against
// the oracle through the library; this program only counts and times it.  It
// fails if a wait of the launch gave up (the device error flag).
//
// usage: layer_counters [shape 8b|1b] [context 1142] [copies 2]
#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>

#include "pard_internal.h"

using namespace pard;

#define CHECK(x)                                                                    \
  do {                                                                              \
    hipError_t e_ = (x);                                                            \
    if (e_ != hipSuccess) {                                                         \
      fprintf(stderr, "%s failed: %s\n", #x, hipGetErrorString(e_));                \
      return 1;                                                                     \
    }                                                                               \
  } while (0)

// fp16 values in about [-1/32, 1/32) from a 32-bit integer hash of the index.
__global__ void k_fill_f16(uint16_t* p, size_t n, uint32_t seed) {
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x) {
    uint32_t h = (uint32_t)i * 0x9E3779B1u ^ seed;
    h ^= h >> 15; h *= 0x2C1B3C6Du; h ^= h >> 12; h *= 0x297A2D39u; h ^= h >> 15;
    p[i] = f16_bits(((float)(h >> 8) * (1.0f / 16777216.0f) - 0.5f) * (1.0f / 16.0f));
  }
}

__global__ void k_fill_value(float* p, size_t n, float v) {
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x) p[i] = v;
}

struct Shape {
  const char* name;
  int d, n_heads, n_kv, hd, ffn;
  int rows, plan_rows;      // rows of the pass; rows its attention plan covers
  int S_q, S_gu, d_split;   // QKV and gate/up strips per tile; down input ranges
};

int main(int argc, char** argv) {
  const char* which = argc > 1 ? argv[1] : "8b";
  const int context = argc > 2 ? atoi(argv[2]) : 1142;
  const int copies = argc > 3 ? atoi(argv[3]) : 2;
  const Shape sh = strcmp(which, "1b") == 0 ? Shape{"1B draft layer", 2048, 32, 8, 64, 8192, 8, 16, 1, 4, 2}
                                            : Shape{"8B target layer", 4096, 32, 8, 128, 14336, 9, 9, 2, 7, 1};
  constexpr int kCap = kAttnWideMaxKeys;
  if ((strcmp(which, "8b") != 0 && strcmp(which, "1b") != 0) || context < 0 || context + sh.plan_rows > kCap ||
      copies < 1 || copies > 8) {
    fprintf(stderr, "usage: layer_counters [8b|1b] [context 0..%d] [copies 1..8]\n", kCap - sh.plan_rows);
    return 2;
  }
  const int pos0 = context;
  const int d = sh.d, hd = sh.hd, q_dim = sh.n_heads * hd, kv_dim = sh.n_kv * hd;
  const int f_pad = (sh.ffn + 31) / 32 * 32;
  // tile plans (as the engine's for these shapes)
  const int q_strips = (q_dim + 2 * kv_dim) / 16, q_tiles = q_strips / sh.S_q, kb_d = d / 32;
  const int group = sh.n_heads / sh.n_kv;
  const int n_qblocks = (sh.plan_rows * group + 15) / 16, n_attn = sh.n_kv * n_qblocks;
  const int l_bound = pos0 + sh.plan_rows, split_len = (l_bound + 127) / 128 * 128;
  const int o_strips = d / 16, kb_o = q_dim / 32;
  const int gu_strips = 2 * f_pad / 16, gu_tiles = gu_strips / sh.S_gu;
  const int d_strips = d / 16, kb_f = f_pad / 32, d_units = d_strips * sh.d_split;
  const int cap_o = qkv_attn_capacity(1, sh.S_q, hd, kb_o);
  const int o_extra0 = std::max(0, std::min(cap_o - q_tiles - n_attn, o_strips - q_tiles));
  const int pre = std::min(qkv_attn_gu_pre_max(sh.S_q, hd, kb_o, sh.S_gu, 1), kb_d / 4);
  const int cap = pre >= 1 ? qkv_attn_capacity(1, sh.S_q, hd, kb_o, sh.S_gu, pre, 1) : 0;
  const int o_extra = std::max({o_extra0, gu_tiles - q_tiles - n_attn, d_units - q_tiles - n_attn});
  const int o_two = std::max(0, o_strips - q_tiles - o_extra);
  const int grid = q_tiles + n_attn + o_extra;
  if (q_strips % sh.S_q || gu_strips % sh.S_gu || cap_o < q_tiles + n_attn || cap <= 0 || gu_tiles > cap ||
      grid > cap || o_two > o_extra) {
    fprintf(stderr, "plan does not fit: grid %d of %d, o_two %d, o_extra %d, gate/up preload %d\n", grid, cap, o_two,
            o_extra, pre);
    return 2;
  }

  // weights, `copies` sets
  const size_t wq = (size_t)q_strips * kb_d * 512, wo = (size_t)o_strips * kb_o * 512;
  const size_t wgu = (size_t)gu_strips * kb_d * 512, wd = (size_t)d_strips * kb_f * 512;
  const size_t w_layer = wq + wo + wgu + wd;
  uint16_t* W;
  CHECK(hipMalloc(&W, w_layer * 2 * copies));
  k_fill_f16<<<2048, 256>>>(W, w_layer * copies, 1u);
  // activations, cache, descriptor, counters
  uint16_t *xg, *q, *attn, *h, *kc, *vc;
  float *ss, *x, *g, *part;
  float2* rope;
  int *cnt, *err, *split_cnt, *ovf;
  FwdDesc* desc;
  const int ss_stride = std::max(o_strips, 1);
  CHECK(hipMalloc(&xg, sizeof(uint16_t) * kMaxRows * d));
  CHECK(hipMalloc(&q, sizeof(uint16_t) * kMaxPassRows * q_dim));
  CHECK(hipMalloc(&attn, sizeof(uint16_t) * kMaxPassRows * q_dim));
  CHECK(hipMalloc(&h, sizeof(uint16_t) * kMaxRows * f_pad));
  CHECK(hipMalloc(&kc, sizeof(uint16_t) * kv_dim * kCap));
  CHECK(hipMalloc(&vc, sizeof(uint16_t) * kv_dim * kCap));
  CHECK(hipMalloc(&ss, sizeof(float) * kMaxPassRows * ss_stride));
  CHECK(hipMalloc(&x, sizeof(float) * kMaxRows * d));
  CHECK(hipMalloc(&g, sizeof(float) * d));
  CHECK(hipMalloc(&part, sizeof(float) * kSplitPartFloats));
  CHECK(hipMalloc(&rope, sizeof(float2) * kCap * hd / 2));
  CHECK(hipMalloc(&cnt, sizeof(int) * kFuseInts));
  CHECK(hipMalloc(&err, sizeof(int) * 64));
  CHECK(hipMalloc(&split_cnt, sizeof(int) * kSplitCounters));
  CHECK(hipMalloc(&ovf, sizeof(int)));
  CHECK(hipMalloc(&desc, sizeof(FwdDesc)));
  k_fill_f16<<<256, 256>>>(xg, (size_t)kMaxRows * d, 2u);
  k_fill_f16<<<256, 256>>>(kc, (size_t)kv_dim * kCap, 3u);
  k_fill_f16<<<256, 256>>>(vc, (size_t)kv_dim * kCap, 4u);
  k_fill_value<<<256, 256>>>(ss, (size_t)kMaxPassRows * ss_stride, (float)d / 3072.0f / o_strips);
  k_fill_value<<<256, 256>>>(x, (size_t)kMaxRows * d, 0.5f);
  k_fill_value<<<64, 256>>>(g, d, 1.0f);
  k_fill_value<<<256, 256>>>(reinterpret_cast<float*>(rope), (size_t)kCap * hd, 0.5f);
  CHECK(hipGetLastError());
  CHECK(hipMemset(err, 0, sizeof(int) * 64));
  CHECK(hipMemset(split_cnt, 0, sizeof(int) * kSplitCounters));
  CHECK(hipMemset(ovf, 0, sizeof(int)));
  static FwdDesc hdsc;
  hdsc.n_rows = sh.rows;
  hdsc.n_seq = 1;
  hdsc.seq[0] = PassSeq{0, 0, sh.rows, sh.rows, pos0, 0, 0, 0};
  for (int r = 0; r < sh.rows; ++r) {
    hdsc.pos[r] = pos0 + r;
    hdsc.slot[r] = 0;
  }
  CHECK(hipMemcpy(desc, &hdsc, sizeof hdsc, hipMemcpyHostToDevice));

  // the launch's arguments, as the engine's forward() builds them
  GemmArgs qa{}, oa{}, ga{}, da{};
  for (GemmArgs* a : {&qa, &oa, &ga, &da}) {
    a->act_rows = kMaxRows;
    a->desc = desc;
    a->eps = 1e-5f;
    a->inv_k = 1.0f / d;
    a->ss_stride = ss_stride;
    a->ovf = ovf;
    a->ksplit = 1;
  }
  qa.kb_total = kb_d; qa.n_strips = q_strips; qa.n_tiles = q_tiles; qa.kb_split = kb_d;
  qa.A = xg; qa.lda = d; qa.ss_in = ss; qa.ss_tiles = o_strips; qa.out = q; qa.ld_out = q_dim;
  qa.kc = kc; qa.vc = vc; qa.cap = kCap; qa.kv_seq_stride = (size_t)kv_dim * kCap; qa.rope = rope;
  qa.q_dim = q_dim; qa.kv_dim = kv_dim; qa.hd = hd;
  oa.kb_total = kb_o; oa.n_strips = o_strips; oa.n_tiles = o_strips; oa.kb_split = kb_o;
  oa.A = attn; oa.lda = q_dim; oa.x = x; oa.ldx = d; oa.g_next = g; oa.xg = xg; oa.ss_out = ss;
  ga.kb_total = kb_d; ga.n_strips = gu_strips; ga.n_tiles = gu_tiles; ga.kb_split = kb_d;
  ga.A = xg; ga.lda = d; ga.ss_in = ss; ga.ss_tiles = o_strips; ga.out = h;
  da.kb_total = kb_f; da.n_strips = d_strips; da.n_tiles = d_strips; da.ksplit = sh.d_split;
  da.kb_split = (kb_f + sh.d_split - 1) / sh.d_split; da.part = part; da.counters = split_cnt;
  da.A = h; da.lda = f_pad; da.x = x; da.ldx = d; da.g_next = g; da.xg = xg; da.ss_out = ss;
  AttnArgs aa{};
  aa.q = q; aa.ldq = q_dim; aa.kc = kc; aa.vc = vc; aa.kv_seq_stride = (size_t)kv_dim * kCap; aa.cap = kCap;
  aa.out = attn; aa.act_rows = kMaxRows; aa.desc = desc; aa.n_heads = sh.n_heads; aa.n_kv = sh.n_kv;
  aa.nqt = 1; aa.n_qblocks = n_qblocks; aa.split_len = split_len; aa.n_splits = 1; aa.n_seq = 1;
  aa.scale = 1.0f / sqrtf((float)hd); aa.part = part; aa.wide = 1;
  FuseCtl f{};
  f.counters = cnt; f.err = err; f.n_prod = q_tiles; f.n_cons = n_attn;
  f.o_units = o_strips; f.o_extra = o_extra; f.o_two = o_two;
  f.gu_tiles = gu_tiles; f.gu_pre = pre; f.gu_pre_q = pre;
  f.n_odone = std::min(q_tiles + o_extra, o_strips - o_two);
  f.d_tiles = d_units;

  hipEvent_t e0, e1;
  CHECK(hipEventCreate(&e0));
  CHECK(hipEventCreate(&e1));
  int launch = 0;
  auto run = [&]() {
    uint16_t* w = W + w_layer * (launch++ % copies);
    qa.W = w; oa.W = w + wq; ga.W = w + wq + wo; da.W = w + wq + wo + wgu;
    hipError_t e = hipMemsetAsync(cnt, 0, sizeof(int) * kFuseInts, 0);
    if (e != hipSuccess) return e;
    return launch_qkv_attn(1, sh.S_q, hd, qa, aa, f, &oa, &ga, sh.S_gu, &da, 0);
  };
  for (int i = 0; i < 20; ++i) CHECK(run());
  CHECK(hipDeviceSynchronize());
  const int n = 100;
  double ms = 0.0;
  for (int i = 0; i < n; ++i) {
    uint16_t* w = W + w_layer * (launch++ % copies);
    qa.W = w; oa.W = w + wq; ga.W = w + wq + wo; da.W = w + wq + wo + wgu;
    CHECK(hipMemsetAsync(cnt, 0, sizeof(int) * kFuseInts, 0));
    CHECK(hipEventRecord(e0, 0));
    CHECK(launch_qkv_attn(1, sh.S_q, hd, qa, aa, f, &oa, &ga, sh.S_gu, &da, 0));
    CHECK(hipEventRecord(e1, 0));
    CHECK(hipEventSynchronize(e1));
    float t = 0.f;
    CHECK(hipEventElapsedTime(&t, e0, e1));
    ms += t;
  }
  int h_err = 0;
  CHECK(hipMemcpy(&h_err, err, sizeof(int), hipMemcpyDeviceToHost));
  const double us = ms * 1e3 / n;
  const double wbytes = (double)w_layer * 2;
  printf("%s: %d workgroups (%d QKV tiles, %d attention, %d extra), gate/up preload %d iterations, "
         "context %d, %d weight copies: %.2f us per launch, weights %.1f MB, %.2f TB/s\n",
         sh.name, grid, q_tiles, n_attn, o_extra, pre, context, copies, us, wbytes / 1e6, wbytes / (us * 1e-6) / 1e12);
  if (h_err) {
    fprintf(stderr, "a wait of the launch exceeded its spin limit: the launch's plan is inconsistent\n");
    return 3;
  }
  CHECK(hipFree(W)); CHECK(hipFree(xg)); CHECK(hipFree(q)); CHECK(hipFree(attn)); CHECK(hipFree(h));
  CHECK(hipFree(kc)); CHECK(hipFree(vc)); CHECK(hipFree(ss)); CHECK(hipFree(x)); CHECK(hipFree(g));
  CHECK(hipFree(part)); CHECK(hipFree(rope)); CHECK(hipFree(cnt)); CHECK(hipFree(err)); CHECK(hipFree(split_cnt));
  CHECK(hipFree(ovf)); CHECK(hipFree(desc));
  return 0;
}
