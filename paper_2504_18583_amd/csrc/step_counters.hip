// Decode steps of the benchmark pair through the library's C ABI alone, for
// hardware counters over whole steps.
//
// Loads the LLaMA3.1-8B target / LLaMA3.2-1B draft pair of the benchmark
// (seeded synthetic weights, seed 1, batch 1), prefills one sequence with a
// fixed 512-token synthetic prompt, runs 4 warm-up steps of the fused decode
// loop (pard_generate, K = 8), launches the marker kernel k_step_marker, and
// runs `steps` more steps.  The dispatches after the marker are exactly the
// measured steps' (the counter summary sums over them:
// profile_summary window --after k_step_marker).  The process loads only the
// library and the HIP runtime it links against.  Prints the measured steps'
// device time per step from pard_stats.
//
// usage: step_counters [steps 16, at most 128]
#include <hip/hip_runtime.h>

#include <cstdio>
#include <cstdlib>
#include <vector>

#include "pard.h"

__global__ void k_step_marker(int* p) {
  if (threadIdx.x == 0 && p) p[0] = 0;
}

namespace {

pard_model_spec llama(int n_layers, int d, int ffn, int hd, int tied, unsigned stream) {
  pard_model_spec s{};
  s.n_layers = n_layers;
  s.d_model = d;
  s.n_heads = 32;
  s.n_kv_heads = 8;
  s.head_dim = hd;
  s.ffn_dim = ffn;
  s.vocab = 128256;
  s.rms_eps = 1e-5f;
  s.rope_theta = 5e5f;
  s.init_std = 0.02f;
  s.tied_embeddings = tied;
  s.dtype = PARD_BF16;
  s.weight_stream = stream;
  s.seed = 1;
  return s;
}

int fail(const char* what, int code) {
  fprintf(stderr, "%s failed: %d\n", what, code);
  return 1;
}

}  // namespace

int main(int argc, char** argv) {
  const int steps = argc > 1 ? atoi(argv[1]) : 16;
  if (steps < 1 || steps > 128) {
    fprintf(stderr, "usage: step_counters [steps 1..128]\n");
    return 2;
  }
  const pard_model_spec t = llama(32, 4096, 14336, 128, 0, 0), d = llama(16, 2048, 8192, 64, 1, 1);
  const int max_ctx = 2048, max_k = 8, k = 8, prompt_len = 512;
  const size_t bytes = pard_arena_bytes(&t, &d, 1, max_ctx, max_k);
  if (bytes == 0) return fail("pard_arena_bytes", 0);
  void* arena = nullptr;
  hipStream_t st = nullptr;
  int* flag = nullptr;
  if (hipMalloc(&arena, bytes) != hipSuccess || hipStreamCreate(&st) != hipSuccess ||
      hipMalloc(&flag, sizeof(int)) != hipSuccess)
    return fail("device allocation", 0);
  pard_ctx* c = nullptr;
  int r = pard_model_load(&t, &d, t.vocab - 1, 1, max_ctx, max_k, arena, bytes, st, &c);
  if (r != PARD_OK) return fail("pard_model_load", r);
  std::vector<int32_t> prompt(prompt_len);
  for (int i = 0; i < prompt_len; ++i) prompt[i] = (int32_t)((i * 7919u + 13u) % (unsigned)(t.vocab - 1));
  int32_t first = 0;
  if ((r = pard_prefill(c, 0, prompt.data(), prompt_len, &first)) != PARD_OK) return fail("pard_prefill", r);
  const int32_t seq = 0;
  // at most K + 1 tokens per step: the KV stays within max_ctx
  std::vector<int32_t> out((size_t)(steps + 4) * (k + 1) + 1);
  pard_stats s{};
  if ((r = pard_generate(c, 1, &seq, k, (int32_t)out.size(), 4, out.data(), &s)) != PARD_OK)
    return fail("pard_generate (warm-up)", r);
  k_step_marker<<<1, 64, 0, st>>>(flag);
  if (hipGetLastError() != hipSuccess) return fail("marker launch", 0);
  if ((r = pard_generate(c, 1, &seq, k, (int32_t)out.size(), steps, out.data(), &s)) != PARD_OK)
    return fail("pard_generate", r);
  if (hipStreamSynchronize(st) != hipSuccess) return fail("hipStreamSynchronize", 0);
  printf("8B/1B K=%d: %lld measured steps, %.4f ms per step (device clock), %lld tokens\n", k, (long long)s.steps,
         s.steps > 0 ? s.elapsed_ms / (double)s.steps : 0.0, (long long)s.tokens);
  pard_free(c);
  (void)hipFree(flag);
  (void)hipFree(arena);
  (void)hipStreamDestroy(st);
  return s.steps == steps ? 0 : 3;
}
