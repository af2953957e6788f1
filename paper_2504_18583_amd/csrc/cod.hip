// Conditional drop-token (COD) training-data processing (Sec. 3.2 eqs. 9-11,
// Alg. 1, App. B), one workgroup per sample.
//
// A sample of L tokens has n = L - 1 columns per subtask k = 1..K.  Subtask 1
// keeps every column (the real tokens).  Column j of subtask k >= 2 (a mask
// token at position j, label t_{j+1}) may be kept only if its whole context
// is kept -- j >= k - 1 and column j - 1 of subtask k - 1 kept -- and the
// subtask keeps min(#valid, floor(n * gamma_k + 1/2)) of the valid columns,
// gamma_k = max(r^{k-1}, r_min): those with the smallest (key, j), key a
// 24-bit SplitMix64 value of (seed, sample, k, j).  The kept columns of all
// subtasks are packed in subtask order, each in column order.
//
// Per subtask the workgroup marks the valid columns (LDS flags), counts them,
// sorts (key, column) pairs with a bitonic sort in LDS when only some are
// kept, and writes the kept columns through a block-wide exclusive scan.  The
// sort is barrier-bound, so workgroups are small (256 threads) and their LDS
// is sized to the batch's longest sample: several workgroups share a CU and
// overlap their barrier waits.
// Only integers and the float64 keep count decide anything, so results are
// bit-exact and independent of timing.
#include "pard_internal.h"

namespace pard {
namespace {

constexpr int kCodThreads = 256;
constexpr int kCodSort = 8192;            // largest bitonic sort (a power of two >= the columns)

__device__ __forceinline__ int wave_excl_scan_int(int v, int lane, int* total) {
  int x = v;
  for (int off = 1; off < 64; off <<= 1) {
    const int o = __shfl_up(x, off);
    if (lane >= off) x += o;
  }
  *total = __shfl(x, 63);
  return x - v;
}

// Exclusive scan of one count per thread over the workgroup (thread order).
__device__ int block_excl_scan(int v, int* wave_s, int* total) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  int wt;
  const int ex = wave_excl_scan_int(v, lane, &wt);
  if (lane == 0) wave_s[wave] = wt;
  __syncthreads();
  int base = 0, all = 0;
  for (int w = 0; w < kCodThreads / 64; ++w) {
    if (w < wave) base += wave_s[w];
    all += wave_s[w];
  }
  __syncthreads();                                 // wave_s is reused by the next call
  *total = all;
  return base + ex;
}

__global__ __launch_bounds__(kCodThreads) void k_cod(const int32_t* __restrict__ tokens, const int64_t* tok_off,
                                                      const int64_t* out_off, CodArgs a, int p_max) {
  // dynamic LDS: sort_s [p_max] (64-bit), then prev_s and cur_s [p_max] (bytes)
  extern __shared__ uint64_t sort_s[];
  uint8_t* prev_s = reinterpret_cast<uint8_t*>(sort_s + p_max);
  uint8_t* cur_s = prev_s + p_max;
  __shared__ int wave_s[kCodThreads / 64];
  __shared__ int count_s;
  const int s = blockIdx.x, tid = threadIdx.x;
  const int64_t t0 = tok_off[s];
  const int n = (int)(tok_off[s + 1] - t0) - 1;     // columns; the host checked 1 <= n <= kCodSort
  const int32_t* t = tokens + t0;
  const int64_t o0 = out_off[s];
  int written = 0;
  // subtask 1: every real token
  for (int j = tid; j < n; j += kCodThreads) {
    a.ids[o0 + j] = t[j];
    a.labels[o0 + j] = t[j + 1];
    a.pos[o0 + j] = j;
    a.section[o0 + j] = 1;
    a.column[o0 + j] = j;
    prev_s[j] = 1;
  }
  written = n;
  const uint64_t z_sample = mix64(a.seed + ((uint64_t)s + 1) * kGamma);
  double gamma = 1.0;
  for (int k = 2; k <= a.k_max; ++k) {
    gamma *= a.r;
    const int target = (int)floor((double)n * fmax(gamma, a.r_min) + 0.5);
    const uint64_t z_k = mix64(z_sample + ((uint64_t)k + 1) * kGamma);
    if (tid == 0) count_s = 0;
    __syncthreads();
    // valid columns: a real token before them and the previous mask on their diagonal kept
    int mine = 0;
    for (int j = tid; j < n; j += kCodThreads) {
      const uint8_t v = (j >= k - 1 && prev_s[j - 1]) ? 1 : 0;
      cur_s[j] = v;
      mine += v;
    }
    if (mine) atomicAdd(&count_s, mine);
    __syncthreads();
    const int n_valid = count_s;
    const int keep = min(n_valid, target);
    if (keep < n_valid) {
      // the `keep` valid columns with the smallest (key, column)
      int P = 1;
      while (P < n) P <<= 1;
      for (int j = tid; j < P; j += kCodThreads) {
        uint64_t e = ~0ull;
        if (j < n && cur_s[j]) e = ((mix64(z_k + ((uint64_t)j + 1) * kGamma) >> 40) << 32) | (uint32_t)j;
        sort_s[j] = e;
      }
      __syncthreads();
      for (int size = 2; size <= P; size <<= 1) {
        for (int stride = size >> 1; stride > 0; stride >>= 1) {
          for (int i = tid; i < P / 2; i += kCodThreads) {
            const int lo = 2 * i - (i & (stride - 1)), hi = lo + stride;
            const bool up = (lo & size) == 0;
            const uint64_t x = sort_s[lo], y = sort_s[hi];
            if ((x > y) == up) { sort_s[lo] = y; sort_s[hi] = x; }
          }
          __syncthreads();
        }
      }
      for (int j = tid; j < n; j += kCodThreads) cur_s[j] = 0;
      __syncthreads();
      for (int i = tid; i < keep; i += kCodThreads) cur_s[(uint32_t)sort_s[i]] = 1;
      __syncthreads();
    }
    // pack the kept columns in column order: thread t owns columns [t*per, (t+1)*per)
    const int per = (n + kCodThreads - 1) / kCodThreads;
    const int c0 = min(tid * per, n), c1 = min(c0 + per, n);
    int cnt = 0;
    for (int j = c0; j < c1; ++j) cnt += cur_s[j];
    int total;
    int at = written + block_excl_scan(cnt, wave_s, &total);
    for (int j = c0; j < c1; ++j) {
      if (!cur_s[j]) continue;
      a.ids[o0 + at] = a.mask_id;
      a.labels[o0 + at] = t[j + 1];
      a.pos[o0 + at] = j;
      a.section[o0 + at] = k;
      a.column[o0 + at] = j;
      ++at;
    }
    written += total;
    __syncthreads();
    for (int j = tid; j < n; j += kCodThreads) prev_s[j] = cur_s[j];
    __syncthreads();
  }
  if (tid == 0) a.out_len[s] = written;
}

}  // namespace

int cod_max_columns() { return kCodSort; }

hipError_t launch_cod(const int32_t* tokens, const int64_t* tok_off, const int64_t* out_off, int n_samples,
                      int max_columns, const CodArgs& a, hipStream_t st) {
  if (n_samples < 1 || a.k_max < 1 || max_columns < 1 || max_columns > kCodSort) return hipErrorInvalidValue;
  int p_max = 1;
  while (p_max < max_columns) p_max <<= 1;
  const size_t lds = (size_t)p_max * (sizeof(uint64_t) + 2);
  k_cod<<<n_samples, kCodThreads, lds, st>>>(tokens, tok_off, out_off, a, p_max);
  return hipGetLastError();
}

}  // namespace pard
