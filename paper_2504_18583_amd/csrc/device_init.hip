// Load-time kernels: seeded weight generation straight into the strip-packed
// layout (each bf16 weight kept in fp16 encoding), rotary tables, fills; and
// the per-pass embedding gather.
#include "device_init.h"

namespace pard {
namespace {

__device__ __forceinline__ uint16_t f2bf(float f) {
  const uint32_t u = __float_as_uint(f);
  return (uint16_t)((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
}

// Box-Muller pair j of the stream `key`: elements 2j (cosine) and 2j+1 (sine).
__device__ __forceinline__ void normal_pair(uint64_t key, uint64_t j, double* n0, double* n1) {
  const uint64_t z0 = mix64(key + (2 * j + 1) * kGamma);
  const uint64_t z1 = mix64(key + (2 * j + 2) * kGamma);
  const double u1 = (double)((z0 >> 11) + 1) * 0x1.0p-53;
  const double u2 = (double)(z1 >> 11) * 0x1.0p-53;
  const double r = sqrt(-2.0 * log(u1));
  const double th = 6.283185307179586 * u2;
  *n0 = r * cos(th);
  *n1 = r * sin(th);
}

// bf16 value of the weight (the model's parameter)
__device__ __forceinline__ uint16_t weight_bits(double n, double stdv) {
  return f2bf((float)(n * stdv));
}

// The same value in the fp16 encoding the GEMMs read (exact when |w| >= 2^-14;
// smaller weights round to the nearest fp16 subnormal, within 2^-25).
__device__ __forceinline__ uint16_t weight_f16(double n, double stdv) {
  return f16_bits(__uint_as_float((uint32_t)weight_bits(n, stdv) << 16));
}

// Canonical (tensor, row) of packed row `n`; false for padding rows.
__device__ __forceinline__ bool map_row(const GenArgs& a, int n, uint64_t* key, int* row) {
  if (a.map == MAP_IDENTITY) {
    if (n >= a.rows) return false;
    *key = a.key0;
    *row = n;
    return true;
  }
  if (a.map == MAP_QKV) {
    const int hd = a.hd;
    if (n < a.q_dim + a.kv_dim) {
      const bool is_q = n < a.q_dim;
      const int p = is_q ? n : n - a.q_dim;
      const int head = p / hd, j = p % hd;
      *row = head * hd + ((j & 1) ? (j >> 1) + hd / 2 : (j >> 1));
      *key = is_q ? a.key0 : a.key1;
      return true;
    }
    if (n < a.q_dim + 2 * a.kv_dim) {
      *row = n - a.q_dim - a.kv_dim;
      *key = a.key2;
      return true;
    }
    return false;
  }
  // MAP_GATEUP: every strip holds 8 gate rows then the 8 up rows of the same
  // features
  const int c = n & 15;
  const int r = (n >> 4) * 8 + (c & 7);
  if (r >= a.rows) return false;
  *row = r;
  *key = (c & 8) ? a.key1 : a.key0;
  return true;
}

// One thread per (strip, k-block, lane): 8 bf16 = 4 Box-Muller pairs.
__global__ void k_gen_packed(const GenArgs a) {
  const size_t total = (size_t)a.n_strips * a.kb_total * 64;
  for (size_t t = (size_t)blockIdx.x * blockDim.x + threadIdx.x; t < total;
       t += (size_t)gridDim.x * blockDim.x) {
    const int lane = (int)(t & 63);
    const size_t blk = t >> 6;
    const int strip = (int)(blk % a.n_strips);   // k-block-major: (kb, strip) blocks
    const int kb = (int)(blk / a.n_strips);
    const int n = strip * 16 + (lane & 15);
    const int k0 = kb * 32 + (lane >> 4) * 8;
    uint16_t out[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    uint64_t key;
    int row;
    if (map_row(a, n, &key, &row)) {
      for (int e = 0; e < 8; e += 2) {
        const int k = k0 + e;
        if (k >= a.cols) break;
        const uint64_t idx = (uint64_t)row * a.cols + k;   // even: cols is even
        double n0, n1;
        normal_pair(key, idx >> 1, &n0, &n1);
        out[e] = weight_f16(n0, a.stdv);
        out[e + 1] = weight_f16(n1, a.stdv);
      }
    }
    uint4 v;
    v.x = out[0] | ((uint32_t)out[1] << 16);
    v.y = out[2] | ((uint32_t)out[3] << 16);
    v.z = out[4] | ((uint32_t)out[5] << 16);
    v.w = out[6] | ((uint32_t)out[7] << 16);
    reinterpret_cast<uint4*>(a.dst)[t] = v;
  }
}

// Bias in packed row order, bf16-rounded values kept as fp32.
__global__ void k_gen_bias(const GenArgs a, float* dst, int n_total) {
  const int n = blockIdx.x * blockDim.x + threadIdx.x;
  if (n >= n_total) return;
  uint64_t key;
  int row;
  float val = 0.f;
  if (map_row(a, n, &key, &row)) {
    double n0, n1;
    normal_pair(key, (uint64_t)row >> 1, &n0, &n1);
    const uint16_t b = weight_bits((row & 1) ? n1 : n0, a.stdv);
    val = __uint_as_float((uint32_t)b << 16);
  }
  dst[n] = val;
}

__global__ void k_fill_f32(float* p, size_t n, float v) {
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x) p[i] = v;
}

__global__ void k_fill_u32(uint32_t* p, size_t n, uint32_t v) {
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += (size_t)gridDim.x * blockDim.x) p[i] = v;
}

// cos/sin of position * theta^(-2i/hd), evaluated in double, stored fp32.
// cos/sin of pos * w_i, w_i = theta^(-2i/hd), optionally with LLaMA-3.1-style
// frequency scaling: wavelengths 2 pi / w below orig / high are kept, above
// orig / low divided by factor, blended in between.
__global__ void k_rope_table(float2* tab, int cap, int hd, double theta, RopeScaling sc) {
  const int half = hd / 2;
  const size_t total = (size_t)cap * half;
  for (size_t t = (size_t)blockIdx.x * blockDim.x + threadIdx.x; t < total; t += (size_t)gridDim.x * blockDim.x) {
    const int pos = (int)(t / half), i = (int)(t % half);
    double inv_freq = pow(theta, -(2.0 * i) / hd);
    if (sc.factor > 0.0) {
      const double wavelen = 6.283185307179586 / inv_freq;
      if (wavelen > sc.orig / sc.low) {
        inv_freq = inv_freq / sc.factor;
      } else if (!(wavelen < sc.orig / sc.high)) {
        const double s = (sc.orig / wavelen - sc.low) / (sc.high - sc.low);
        inv_freq = (1.0 - s) * inv_freq / sc.factor + s * inv_freq;
      }
    }
    const double ang = (double)pos * inv_freq;
    tab[t] = make_float2((float)cos(ang), (float)sin(ang));
  }
}

// x[r, :] = E[ids[r], :] (fp32) from the strip-packed embedding, plus the
// first normalised GEMM's operand xg = fp16(x * g) and the row's sum of squares.
__global__ __launch_bounds__(256) void k_embed(const uint16_t* E, int n_strips, int d, const FwdDesc* desc,
                                               float* x, const float* g, uint16_t* xg, int act_rows, float* ss,
                                               int ss_stride, unsigned long long* t_start, int* fuse_cnt,
                                               int n_sets, int* ovf) {
  __shared__ float wsum[4];
  const int r = blockIdx.x;
  if (r == 0 && threadIdx.x == 0 && t_start) *t_start = wall_clock64();
  // the pass's fused-launch counters start at zero (their last use was in an
  // earlier launch)
  if (r == 0 && fuse_cnt) {
    constexpr int per = kFuseInts / kFuseStride;   // counters per set
    for (int i = threadIdx.x; i < n_sets * per; i += blockDim.x)
      __hip_atomic_store(fuse_cnt + (size_t)(i / per) * kFuseInts + (i % per) * kFuseStride, 0, __ATOMIC_RELAXED,
                         __HIP_MEMORY_SCOPE_AGENT);
  }
  if (r >= desc->n_rows) return;
  const int id = desc->ids[r];
  const size_t strip = (size_t)(id >> 4);
  float sq = 0.f;
  bool bad = false;
  for (int c8 = threadIdx.x; c8 < d / 8; c8 += blockDim.x) {
    const int k0 = c8 * 8, kb = k0 >> 5;
    const int lane = (id & 15) + 16 * ((k0 & 31) >> 3);
    const uint4 w = *reinterpret_cast<const uint4*>(E + (((size_t)kb * n_strips + strip) * 64 + lane) * 8);
    const uint32_t wv[4] = {w.x, w.y, w.z, w.w};
    float v[8];
    for (int i = 0; i < 4; ++i) {
      v[2 * i] = (float)__builtin_bit_cast(_Float16, (uint16_t)(wv[i] & 0xFFFFu));
      v[2 * i + 1] = (float)__builtin_bit_cast(_Float16, (uint16_t)(wv[i] >> 16));
    }
    float4* dst = reinterpret_cast<float4*>(x + (size_t)r * d + k0);
    dst[0] = make_float4(v[0], v[1], v[2], v[3]);
    dst[1] = make_float4(v[4], v[5], v[6], v[7]);
    uint32_t o[4];
    for (int i = 0; i < 4; ++i) {
      o[i] = (uint32_t)f16_flagged(v[2 * i] * g[k0 + 2 * i], bad) |
             ((uint32_t)f16_flagged(v[2 * i + 1] * g[k0 + 2 * i + 1], bad) << 16);
      sq += v[2 * i] * v[2 * i] + v[2 * i + 1] * v[2 * i + 1];
    }
    *reinterpret_cast<uint4*>(xg + act_index(r, k0, act_rows)) = make_uint4(o[0], o[1], o[2], o[3]);
  }
  flag_range(bad, ovf);
  for (int off = 32; off > 0; off >>= 1) sq += __shfl_xor(sq, off);
  if ((threadIdx.x & 63) == 0) wsum[threadIdx.x >> 6] = sq;
  __syncthreads();
  if (threadIdx.x == 0) ss[(size_t)r * ss_stride] = ((wsum[0] + wsum[1]) + wsum[2]) + wsum[3];
}

__global__ void k_gather_u16(const uint16_t* src, const size_t* idx, int n, float* out) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) out[i] = (float)__builtin_bit_cast(_Float16, src[idx[i]]);
}

int blocks_for(size_t n, int per_block) {
  size_t b = (n + per_block - 1) / per_block;
  if (b > 65535 * 4) b = 65535 * 4;
  return (int)(b ? b : 1);
}

}  // namespace

hipError_t launch_gen_packed(const GenArgs& a, hipStream_t st) {
  const size_t total = (size_t)a.n_strips * a.kb_total * 64;
  k_gen_packed<<<blocks_for(total, 256), 256, 0, st>>>(a);
  return hipGetLastError();
}

hipError_t launch_gen_bias(const GenArgs& a, float* dst, int n_total, hipStream_t st) {
  k_gen_bias<<<(n_total + 255) / 256, 256, 0, st>>>(a, dst, n_total);
  return hipGetLastError();
}

hipError_t launch_fill_f32(float* p, size_t n, float v, hipStream_t st) {
  k_fill_f32<<<blocks_for(n, 256), 256, 0, st>>>(p, n, v);
  return hipGetLastError();
}

hipError_t launch_fill_u32(uint32_t* p, size_t n, uint32_t v, hipStream_t st) {
  k_fill_u32<<<blocks_for(n, 256), 256, 0, st>>>(p, n, v);
  return hipGetLastError();
}

hipError_t launch_rope_table(float2* tab, int cap, int hd, double theta, const RopeScaling& sc, hipStream_t st) {
  k_rope_table<<<blocks_for((size_t)cap * hd / 2, 256), 256, 0, st>>>(tab, cap, hd, theta, sc);
  return hipGetLastError();
}

hipError_t launch_embed(const uint16_t* E, int n_strips, int d, const FwdDesc* desc, float* x, const float* g,
                        uint16_t* xg, int act_rows, float* ss, int ss_stride, int max_rows,
                        unsigned long long* t_start, int* fuse_cnt, int n_sets, int* ovf, hipStream_t st) {
  k_embed<<<max_rows, 256, 0, st>>>(E, n_strips, d, desc, x, g, xg, act_rows, ss, ss_stride, t_start, fuse_cnt,
                                    n_sets, ovf);
  return hipGetLastError();
}

hipError_t launch_gather_u16(const uint16_t* src, const size_t* idx, int n, float* out, hipStream_t st) {
  k_gather_u16<<<(n + 255) / 256, 256, 0, st>>>(src, idx, n, out);
  return hipGetLastError();
}

}  // namespace pard
