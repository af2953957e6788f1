// Stand-alone launches of one skinny GEMM shape, for hardware counters and
// launch-shape timing.
//
// Launches k_gemm<MT=1, S, EPI> (EPI_SWIGLU, EPI_RESID or EPI_QKV) over `rows` decode
// rows of a weight of `strips` 16-column strips x `kb` 32-column k-blocks,
// with the input dimension split into P ranges, 20 times untimed and 100 times
// timed, and prints the mean launch time.  The defaults are the LLaMA3.1-8B
// gate/up GEMM (hidden 4096, intermediate 14336, gate and up stacked: 1792
// strips) as the decode step launches it.  `copies` > 1 cycles the launches
// through that many weight copies, so that a small weight is not served from
// the last-level cache on every launch as it would not be in a decode step.
// Weights and activations are seeded pseudo-random fp16 values.  With check
// = 1 it then runs, for every weight copy in turn, the same launch unsplit and
// split and compares the two outputs (they differ only by summation order), a
// test of the split's partial-tile exchange; the numerics of the kernel itself
// are tested against the oracle through the library.  The QKV epilogue
// writes a grouped-query layout of head_dim 128 (query width 4 x the key
// width) at positions 512.. of one sequence's cache.  `ss_tiles` is the number
// of per-tile sums of squares each row scale adds (256 after the 8B down
// projection).
//
// usage: gemm_counters [rows 9] [S 7] [P 1] [strips 1792] [kb 128] [epi swiglu|resid|qkv] [copies 1] [check 0]
//                      [ss_tiles 1] [wavefronts 4|8] [touch -1|0|2]
#include <cstdio>
#include <cstdlib>
#include <cmath>
#include <cstring>
#include <vector>

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

// Reads n 16-byte words of p with the given buffer cache policy (a stand-in
// for a prefetch into the last-level cache); the XOR of what it read is
// stored only when it equals a value no seeded fill produces.
__global__ void k_touch(const uint16_t* p, size_t n16, int policy, unsigned* sink) {
  const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(p), 0, 0x7fffffff, 0x00020000);
  unsigned x = 0;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n16; i += (size_t)gridDim.x * blockDim.x) {
    const auto v = policy == 2 ? __builtin_amdgcn_raw_buffer_load_b128(rs, (int)(i * 16), 0, 2)
                               : __builtin_amdgcn_raw_buffer_load_b128(rs, (int)(i * 16), 0, 0);
    x ^= v[0] ^ v[1] ^ v[2] ^ v[3];
  }
  if (x == 0x9E3779B9u && sink) *sink = x;
}

__global__ void k_fill_value(float* p, size_t n, float v) {
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x) p[i] = v;
}

int main(int argc, char** argv) {
  const int rows = argc > 1 ? atoi(argv[1]) : 9;
  const int S = argc > 2 ? atoi(argv[2]) : 7;
  const int P = argc > 3 ? atoi(argv[3]) : 1;
  const int n_strips = argc > 4 ? atoi(argv[4]) : 2 * 14336 / 16;
  const int kb_total = argc > 5 ? atoi(argv[5]) : 4096 / 32;
  const bool resid = argc > 6 && strcmp(argv[6], "resid") == 0;
  const bool qkv = argc > 6 && strcmp(argv[6], "qkv") == 0;
  const int copies = argc > 7 ? atoi(argv[7]) : 1;
  const bool check = argc > 8 && atoi(argv[8]) != 0;
  const int ss_tiles = argc > 9 ? atoi(argv[9]) : 1;
  const int nw = argc > 10 ? atoi(argv[10]) : 4;
  // touch >= 0: before each timed launch, read its weight copy with cache
  // policy `touch` (0 default, 2 non-temporal; 10 + policy: read the next
  // copy instead, the control) and time the launch alone
  const int touch = argc > 11 ? atoi(argv[11]) : -1;
  const int epi = resid ? EPI_RESID : qkv ? EPI_QKV : EPI_SWIGLU;
  constexpr int kHd = 128, kCap = 1024, kPos0 = 512;
  const int kb_split = P > 0 ? (kb_total + P - 1) / P : 0;
  const bool wide_s = epi == EPI_SWIGLU && S >= 7 && S <= 10;
  if (rows < 1 || rows > kMaxRows || !(S == 1 || S == 2 || S == 4 || wide_s) ||
      n_strips < 1 || (n_strips % S != 0 && S < 8) || kb_total < 1 || P < 1 || (P - 1) * kb_split >= kb_total || copies < 1 ||
      copies > 64 || (size_t)n_strips * kb_total * 1024 * copies > ((size_t)8 << 30) || ss_tiles < 1 ||
      ss_tiles > n_strips || (qkv && ((n_strips * 16) % (6 * kHd) != 0 || check)) || (nw != 4 && nw != 8)) {
    fprintf(stderr, "bad shape: rows 1..%d, S in {1, 2, 4, 7-10 (swiglu)}, S | strips (S < 8), every input range non-empty, "
            "copies 1..64 of at most 8 GiB in all, 1 <= ss_tiles <= strips; qkv: 6 x 128 | columns, no check; "
            "4 or 8 wavefronts\n",
            kMaxRows);
    return 2;
  }
  const int hidden = kb_total * 32;
  const int out_cols = n_strips * 16;
  const size_t w_elems = (size_t)n_strips * kb_total * 512;
  const size_t a_elems = (size_t)kMaxRows * hidden;
  const size_t o_elems = ((size_t)n_strips * 16 / 32 + 1) * kMaxRows * 32;   // k-blocked rows, one block spare
  uint16_t *W, *A, *out;
  float *ss, *x, *g, *ss_out, *part;
  int* counters;
  FwdDesc* desc;
  uint16_t *kc, *vc;
  float2* rope;
  const int kv_dim = out_cols / 6, q_dim = out_cols - 2 * kv_dim;
  CHECK(hipMalloc(&kc, sizeof(uint16_t) * kv_dim * kCap));
  CHECK(hipMalloc(&vc, sizeof(uint16_t) * kv_dim * kCap));
  CHECK(hipMalloc(&rope, sizeof(float2) * kCap * kHd / 2));
  CHECK(hipMalloc(&W, w_elems * 2 * copies));
  CHECK(hipMalloc(&A, a_elems * 2));
  CHECK(hipMalloc(&out, o_elems * 2));
  const int ss_stride = std::max(ss_tiles, (n_strips + S - 1) / S);   // [row][tile] sums, in and out
  CHECK(hipMalloc(&ss, sizeof(float) * kMaxPassRows * ss_stride));
  CHECK(hipMalloc(&x, sizeof(float) * kMaxRows * out_cols));
  CHECK(hipMalloc(&g, sizeof(float) * out_cols));
  CHECK(hipMalloc(&ss_out, sizeof(float) * (size_t)kMaxPassRows * ss_stride));
  CHECK(hipMalloc(&part, sizeof(float) * kSplitPartFloats));
  CHECK(hipMalloc(&counters, sizeof(int) * kSplitCounters));
  CHECK(hipMalloc(&desc, sizeof(FwdDesc)));
  CHECK(hipMemset(counters, 0, sizeof(int) * kSplitCounters));
  k_fill_f16<<<1024, 256>>>(W, w_elems * copies, 1u);
  k_fill_f16<<<64, 256>>>(A, a_elems, 2u);
  k_fill_value<<<64, 256>>>(ss, (size_t)kMaxPassRows * ss_stride, (float)hidden / 3072.0f / ss_tiles);
  k_fill_value<<<64, 256>>>(reinterpret_cast<float*>(rope), (size_t)kCap * kHd, 0.5f);
  k_fill_value<<<64, 256>>>(x, (size_t)kMaxRows * out_cols, 0.5f);
  k_fill_value<<<64, 256>>>(g, out_cols, 1.0f);
  CHECK(hipGetLastError());
  static FwdDesc hd;
  hd.n_rows = rows;
  hd.n_seq = 1;
  hd.seq[0].n_rows = rows;
  hd.seq[0].n_real = rows;
  for (int r = 0; r < rows; ++r) {
    hd.pos[r] = kPos0 + r;
    hd.slot[r] = 0;
  }
  CHECK(hipMemcpy(desc, &hd, sizeof hd, hipMemcpyHostToDevice));

  GemmArgs a{};
  a.kb_total = kb_total; a.n_strips = n_strips; a.n_tiles = (n_strips + S - 1) / S;
  a.ksplit = P; a.kb_split = kb_split; a.part = part; a.counters = counters;
  a.A = A; a.lda = hidden; a.act_rows = kMaxRows; a.desc = desc;
  a.ss_in = ss; a.ss_tiles = ss_tiles; a.ss_stride = ss_stride; a.eps = 1e-5f; a.inv_k = 1.0f / hidden;
  a.out = out; a.ld_out = out_cols;
  a.x = x; a.ldx = out_cols; a.g_next = g; a.xg = out; a.ss_out = ss_out;
  a.kc = kc; a.vc = vc; a.cap = kCap; a.kv_seq_stride = (size_t)kv_dim * kCap; a.rope = rope;
  a.q_dim = q_dim; a.kv_dim = kv_dim; a.hd = kHd;

  hipEvent_t e0, e1;
  CHECK(hipEventCreate(&e0));
  CHECK(hipEventCreate(&e1));
  int launch = 0;
  auto run = [&]() {
    a.W = W + w_elems * (launch++ % copies);
    return launch_gemm(epi, 1, S, nw, a, 0);
  };
  for (int i = 0; i < 20; ++i) CHECK(run());
  CHECK(hipDeviceSynchronize());
  const int n = 100;
  float ms = 0.f;
  if (touch < 0) {
    CHECK(hipEventRecord(e0, 0));
    for (int i = 0; i < n; ++i) CHECK(run());
    CHECK(hipEventRecord(e1, 0));
    CHECK(hipEventSynchronize(e1));
    CHECK(hipEventElapsedTime(&ms, e0, e1));
  } else {
    for (int i = 0; i < n; ++i) {
      // touch >= 10: the control, which reads another copy (policy touch - 10)
      const int cp = touch >= 10 ? (launch + 1) % copies : launch % copies;
      k_touch<<<1024, 256>>>(W + w_elems * cp, w_elems * 2 / 16, touch % 10, nullptr);
      CHECK(hipEventRecord(e0, 0));
      CHECK(run());
      CHECK(hipEventRecord(e1, 0));
      CHECK(hipEventSynchronize(e1));
      float t = 0.f;
      CHECK(hipEventElapsedTime(&t, e0, e1));
      ms += t;
    }
  }
  const double us = ms * 1e3 / n;
  printf("k_gemm<1, %d, %d> %s, %d strips x %d k-blocks, %d rows, %d x %d workgroups of %d wavefronts, %d weight copies: "
         "%.2f us per launch, weights %.2f TB/s\n", S, epi, resid ? "resid" : qkv ? "qkv" : "swiglu", n_strips, kb_total, rows,
         a.n_tiles, P, nw, copies, us, (double)w_elems * 2 / (us * 1e-6) / 1e12);
  if (check) {
    // unsplit reference and split launch per copy, x reset before each (the
    // residual epilogue updates it in place); outputs compared as fp16
    std::vector<uint16_t> ref(o_elems), got(o_elems);
    GemmArgs r = a;
    r.ksplit = 1;
    r.kb_split = kb_total;
    auto to_f = [](uint16_t b) { return (float)__builtin_bit_cast(_Float16, b); };
    double worst = 0.0;
    long bad = 0, compared = 0;
    for (int c = 0; c < copies; ++c) {
      for (int pass = 0; pass < 2; ++pass) {
        GemmArgs& q = pass == 0 ? r : a;
        q.W = W + w_elems * c;
        k_fill_value<<<64, 256>>>(x, (size_t)kMaxRows * out_cols, 0.5f);
        CHECK(hipMemset(out, 0, o_elems * 2));
        CHECK(launch_gemm(epi, 1, S, nw, q, 0));
        CHECK(hipMemcpy(pass == 0 ? ref.data() : got.data(), out, o_elems * 2, hipMemcpyDeviceToHost));
      }
      const int cols = resid ? out_cols : out_cols / 2;
      for (int row = 0; row < rows; ++row)
        for (int k = 0; k < cols; ++k) {
          const size_t i = ((size_t)(k >> 5) * kMaxRows + row) * 32 + (k & 31);
          const double x0 = to_f(ref[i]), x1 = to_f(got[i]);
          const double d = std::fabs(x1 - x0);
          worst = std::max(worst, d);
          bad += !(d <= 2e-3 + 1e-2 * std::fabs(x0));
          ++compared;
        }
    }
    printf("check split %d vs unsplit over %d copies: %ld of %ld outputs outside 2e-3 + 1e-2|ref|, max |diff| %.3g\n",
           P, copies, bad, compared, worst);
    if (bad) return 3;
  }
  CHECK(hipFree(W)); CHECK(hipFree(A)); CHECK(hipFree(out)); CHECK(hipFree(ss)); CHECK(hipFree(x));
  CHECK(hipFree(g)); CHECK(hipFree(ss_out)); CHECK(hipFree(part)); CHECK(hipFree(counters)); CHECK(hipFree(desc));
  CHECK(hipFree(kc)); CHECK(hipFree(vc)); CHECK(hipFree(rope));
  return 0;
}
