// Stand-alone run of one skinny GEMM launch shape, for hardware counters.
//
// Launches the SwiGLU gate/up GEMM (k_gemm<MT=1, S, EPI_SWIGLU>) at the
// LLaMA3.1-8B shape (hidden 4096, intermediate 14336, gate and up stacked:
// 1792 strips of 16 columns) over `rows` decode rows, 20 times untimed and
// 100 times timed, and prints the mean launch time.  It exists so that
// rocprofv3 --pmc can count the HBM bytes of exactly this kernel in a short
// program of its own.  Weights and activations are seeded pseudo-random fp16
// values; the result is not checked (the parity tests do that through the
// library).
//
// usage: gemm_counters [rows (1..64, default 9)] [strips per workgroup S (1, 2, 4, 7; default 7)]
#include <cstdio>
#include <cstdlib>

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

int main(int argc, char** argv) {
  const int rows = argc > 1 ? atoi(argv[1]) : 9;
  const int S = argc > 2 ? atoi(argv[2]) : 7;
  const int hidden = 4096, n_strips = 2 * 14336 / 16, kb_total = hidden / 32;
  if (rows < 1 || rows > kMaxRows || !(S == 1 || S == 2 || S == 4 || S == 7) || n_strips % S != 0) {
    fprintf(stderr, "rows must be in 1..%d and S one of 1, 2, 4, 7\n", kMaxRows);
    return 2;
  }
  const size_t w_elems = (size_t)n_strips * kb_total * 512;
  const size_t a_elems = (size_t)kMaxRows * hidden;
  const size_t o_elems = (size_t)kMaxRows * n_strips * 8;
  uint16_t *W, *A, *out;
  float* ss;
  FwdDesc* desc;
  CHECK(hipMalloc(&W, w_elems * 2));
  CHECK(hipMalloc(&A, a_elems * 2));
  CHECK(hipMalloc(&out, o_elems * 2));
  CHECK(hipMalloc(&ss, sizeof(float) * kMaxPassRows));
  CHECK(hipMalloc(&desc, sizeof(FwdDesc)));
  k_fill_f16<<<1024, 256>>>(W, w_elems, 1u);
  k_fill_f16<<<64, 256>>>(A, a_elems, 2u);
  CHECK(hipGetLastError());
  static float hs[kMaxPassRows];
  for (float& v : hs) v = (float)hidden / 3072.0f;    // sum of squares of each row: rms ~ 1/sqrt(3072)
  CHECK(hipMemcpy(ss, hs, sizeof hs, hipMemcpyHostToDevice));
  static FwdDesc hd;
  hd.n_rows = rows;
  hd.n_seq = 1;
  hd.seq[0].n_rows = rows;
  hd.seq[0].n_real = rows;
  CHECK(hipMemcpy(desc, &hd, sizeof hd, hipMemcpyHostToDevice));

  GemmArgs a{};
  a.W = W; a.kb_total = kb_total; a.n_strips = n_strips; a.n_tiles = n_strips / S;
  a.A = A; a.lda = hidden; a.act_rows = kMaxRows; a.desc = desc;
  a.ss_in = ss; a.ss_tiles = 1; a.eps = 1e-5f; a.inv_k = 1.0f / hidden;
  a.out = out; a.ld_out = n_strips * 8;

  hipEvent_t e0, e1;
  CHECK(hipEventCreate(&e0));
  CHECK(hipEventCreate(&e1));
  for (int i = 0; i < 20; ++i) CHECK(launch_gemm(EPI_SWIGLU, 1, S, 4, a, 0));
  CHECK(hipDeviceSynchronize());
  const int n = 100;
  CHECK(hipEventRecord(e0, 0));
  for (int i = 0; i < n; ++i) CHECK(launch_gemm(EPI_SWIGLU, 1, S, 4, a, 0));
  CHECK(hipEventRecord(e1, 0));
  CHECK(hipEventSynchronize(e1));
  float ms = 0.f;
  CHECK(hipEventElapsedTime(&ms, e0, e1));
  const double us = ms * 1e3 / n;
  printf("k_gemm<1, %d, 2> gate/up 8B shape, %d rows, %d workgroups: %.2f us per launch, weights %.2f TB/s\n", S,
         rows, n_strips / S, us, (double)w_elems * 2 / (us * 1e-6) / 1e12);
  CHECK(hipFree(W)); CHECK(hipFree(A)); CHECK(hipFree(out)); CHECK(hipFree(ss)); CHECK(hipFree(desc));
  return 0;
}
