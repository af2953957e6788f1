// Attainable MFMA rate of the instructions the GEMMs use, measured on the
// device at hand: the practical ceiling beside the published 2.5 PFLOP/s
// dense fp16 figure.
//
// Every wavefront issues back-to-back v_mfma_f32_16x16x32_f16 (the GEMMs'
// instruction) or v_mfma_f32_32x32x16_f16 on register operands, CH
// independent accumulator chains deep, so nothing but the matrix unit and the
// clock it runs at limits the rate.  Operands are seeded pseudo-random fp16
// values in [-1, 1) (the unit's power draw, and with it the clock, depends on
// the data).  One grid of 256 workgroups (one per CU) with 4 or 8 wavefronts
// each; 100 untimed iterations, then `iters` timed by HIP events.
//
// usage: mfma_peak [iters 20000]
#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <vector>

namespace {

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

#define CHECK(x)                                                                                     \
  do {                                                                                               \
    hipError_t e_ = (x);                                                                             \
    if (e_ != hipSuccess) {                                                                          \
      fprintf(stderr, "%s failed: %s (line %d)\n", #x, hipGetErrorString(e_), __LINE__);             \
      exit(1);                                                                                       \
    }                                                                                                \
  } while (0)

// in: 2 x 64 operand vectors (A then B, one per lane); out: one f32x4 per thread
template <int CH>
__global__ __launch_bounds__(512) void k_mfma16(const f16x8* in, f32x4* out, int iters) {
  const int l = threadIdx.x;
  const f16x8 a = in[l & 63], b = in[64 + (l & 63)];
  f32x4 acc[CH];
#pragma unroll
  for (int c = 0; c < CH; ++c) acc[c] = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int i = 0; i < iters; ++i) {
#pragma unroll
    for (int c = 0; c < CH; ++c) acc[c] = __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, acc[c], 0, 0, 0);
  }
  f32x4 s = acc[0];
#pragma unroll
  for (int c = 1; c < CH; ++c) s += acc[c];
  out[blockIdx.x * blockDim.x + l] = s;
}

template <int CH>
__global__ __launch_bounds__(512) void k_mfma32(const f16x8* in, f32x4* out, int iters) {
  const int l = threadIdx.x;
  const f16x8 a = in[l & 63], b = in[64 + (l & 63)];
  f32x16 acc[CH];
#pragma unroll
  for (int c = 0; c < CH; ++c) acc[c] = f32x16{};
  for (int i = 0; i < iters; ++i) {
#pragma unroll
    for (int c = 0; c < CH; ++c) acc[c] = __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, acc[c], 0, 0, 0);
  }
  f32x4 s = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int c = 0; c < CH; ++c) s += f32x4{acc[c][0], acc[c][1], acc[c][2], acc[c][3]};
  out[blockIdx.x * blockDim.x + l] = s;
}

}  // namespace

int main(int argc, char** argv) {
  const int iters = argc > 1 ? atoi(argv[1]) : 20000;
  if (iters < 1 || iters > 1000000) {
    fprintf(stderr, "usage: mfma_peak [iters 1..1000000]\n");
    return 2;
  }
  constexpr int kGrid = 256, kMaxThreads = 512;
  std::vector<_Float16> host(128 * 8);
  uint64_t st = 0x9E3779B97F4A7C15ull;
  for (auto& v : host) {
    st = st * 6364136223846793005ull + 1442695040888963407ull;
    v = (_Float16)((double)(st >> 40) / (double)(1ull << 24) * 2.0 - 1.0);
  }
  f16x8* in = nullptr;
  f32x4* out = nullptr;
  CHECK(hipMalloc(&in, 128 * sizeof(f16x8)));
  CHECK(hipMalloc(&out, (size_t)kGrid * kMaxThreads * sizeof(f32x4)));
  CHECK(hipMemcpy(in, host.data(), 128 * sizeof(f16x8), hipMemcpyHostToDevice));
  hipEvent_t e0, e1;
  CHECK(hipEventCreate(&e0));
  CHECK(hipEventCreate(&e1));
  auto run = [&](const char* name, auto kern, int threads, double flop_per_mfma, int ch) {
    kern<<<kGrid, threads>>>(in, out, 100);
    CHECK(hipGetLastError());
    CHECK(hipDeviceSynchronize());
    CHECK(hipEventRecord(e0));
    kern<<<kGrid, threads>>>(in, out, iters);
    CHECK(hipGetLastError());
    CHECK(hipEventRecord(e1));
    CHECK(hipEventSynchronize(e1));
    float ms = 0.f;
    CHECK(hipEventElapsedTime(&ms, e0, e1));
    const double flop = (double)kGrid * (threads / 64) * iters * ch * flop_per_mfma;
    printf("%-24s %d wavefronts/CU, %d chains: %8.3f ms  %7.1f TFLOP/s  (%.3f of 2.5 PFLOP/s)\n", name,
           threads / 64, ch, ms, flop / ms / 1e9, flop / ms / 1e9 / 2500.0);
  };
  const double f16 = 16.0 * 16 * 32 * 2, f32 = 32.0 * 32 * 16 * 2;
  run("16x16x32 f16", k_mfma16<4>, 256, f16, 4);
  run("16x16x32 f16", k_mfma16<8>, 256, f16, 8);
  run("16x16x32 f16", k_mfma16<8>, 512, f16, 8);
  run("32x32x16 f16", k_mfma32<2>, 256, f32, 2);
  run("32x32x16 f16", k_mfma32<4>, 256, f32, 4);
  run("32x32x16 f16", k_mfma32<4>, 512, f32, 4);
  CHECK(hipFree(out));
  CHECK(hipFree(in));
  return 0;
}
