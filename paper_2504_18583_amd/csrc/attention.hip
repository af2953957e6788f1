// Grouped-query causal attention of a short block of query rows against the
// contiguous bf16 KV cache (the draft pass with its mask rows, the verify pass,
// and prefill chunks).
//
// Grid: (kv_head, key chunk, query block).  A query block holds kAttnQB
// (row, head-in-group) pairs of one KV head, so the K/V tiles staged in LDS are
// shared by the whole GQA group.  Each workgroup walks its key chunk in
// kAttnSub-key sub-chunks with an online softmax (running max m, sum l,
// unnormalised output o, all fp32), then writes (o, m, l) for its chunk.  The
// last workgroup of a (kv_head, query block) -- device-scope counter,
// self-resetting -- merges the chunks in chunk order: deterministic, no float
// atomics.  Causality is by absolute position: key j is visible to the query at
// position pos0 + row iff j <= pos0 + row (the draft's mask rows are ordinary
// causal rows; Sec. 3.1 eq. 7 conditions candidate k on x_<n and m_0..m_{k-1}).
#include "pard_internal.h"

namespace pard {
namespace {

__device__ __forceinline__ float bf_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }
__device__ __forceinline__ uint16_t f2bf(float f) {
  const uint32_t u = __float_as_uint(f);
  return (uint16_t)((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
}

template <int HD>
__global__ __launch_bounds__(kBlock) void k_attn(const AttnArgs p) {
  constexpr int QB = kAttnQB, SUB = kAttnSub;
  constexpr int HW = HD / 2;            // bf16 pairs per row
  constexpr int ND = HD / 16;           // output dims per thread
  __shared__ float qs[QB][HD + 4];
  __shared__ uint32_t ks[SUB][HW + 1];
  __shared__ uint32_t vs[SUB][HW];
  __shared__ float ps[QB][SUB + 1];
  __shared__ int last_s;

  const int kvh = blockIdx.x, c = blockIdx.y, z = blockIdx.z;
  const int tid = threadIdx.x;
  const int group = p.n_heads / p.n_kv;
  const int n_rows = p.desc->n_rows, pos0 = p.desc->pos0;
  const int L_end = pos0 + n_rows;
  const int n_act = (L_end + p.chunk - 1) / p.chunk;
  const int n_qh = n_rows * group;
  if (c >= n_act || z * QB >= n_qh) return;

  const uint16_t* kc = p.kc + (size_t)kvh * p.cap * HD;
  const uint16_t* vc = p.vc + (size_t)kvh * p.cap * HD;

  const float scale = p.scale;
  for (int e = tid; e < QB * HD; e += kBlock) {
    const int qi = e / HD, dd = e % HD, qh = z * QB + qi;
    float val = 0.f;
    if (qh < n_qh) {
      const int r = qh / group, h = kvh * group + qh % group;
      val = __uint_as_float((uint32_t)p.q[(size_t)r * p.ldq + h * HD + dd] << 16) * scale;
    }
    qs[qi][dd] = val;
  }

  const int qi = tid >> 4, sl = tid & 15;
  const int qh = z * QB + qi;
  const int qpos = (qh < n_qh) ? pos0 + qh / group : -1;
  float m = -INFINITY, l = 0.f;
  float o[ND];
#pragma unroll
  for (int j = 0; j < ND; ++j) o[j] = 0.f;

  const int k_begin = c * p.chunk;
  const int k_end = min(L_end, k_begin + p.chunk);
  for (int kb = k_begin; kb < k_end; kb += SUB) {
    __syncthreads();
    for (int e = tid; e < SUB * (HD / 8); e += kBlock) {
      const int kr = e / (HD / 8), cc = e % (HD / 8), key = kb + kr;
      uint4 kv = make_uint4(0, 0, 0, 0), vv = kv;
      if (key < k_end) {
        kv = *reinterpret_cast<const uint4*>(kc + (size_t)key * HD + cc * 8);
        vv = *reinterpret_cast<const uint4*>(vc + (size_t)key * HD + cc * 8);
      }
      ks[kr][cc * 4 + 0] = kv.x; ks[kr][cc * 4 + 1] = kv.y; ks[kr][cc * 4 + 2] = kv.z; ks[kr][cc * 4 + 3] = kv.w;
      vs[kr][cc * 4 + 0] = vv.x; vs[kr][cc * 4 + 1] = vv.y; vs[kr][cc * 4 + 2] = vv.z; vs[kr][cc * 4 + 3] = vv.w;
    }
    __syncthreads();
    float sc[SUB / 16];
    float mx = -INFINITY;
#pragma unroll
    for (int jj = 0; jj < SUB / 16; ++jj) {
      const int kl = sl + 16 * jj, key = kb + kl;
      float acc = 0.f;
#pragma unroll 8
      for (int d2 = 0; d2 < HW; ++d2) {
        const uint32_t w = ks[kl][d2];
        acc += qs[qi][2 * d2] * bf_lo(w) + qs[qi][2 * d2 + 1] * bf_hi(w);
      }
      sc[jj] = (key < k_end && key <= qpos) ? acc : -INFINITY;
      mx = fmaxf(mx, sc[jj]);
    }
#pragma unroll
    for (int off = 8; off > 0; off >>= 1) mx = fmaxf(mx, __shfl_xor(mx, off));
    const float m_new = fmaxf(m, mx);
    float psum = 0.f;
#pragma unroll
    for (int jj = 0; jj < SUB / 16; ++jj) {
      const float pv = (sc[jj] == -INFINITY) ? 0.f : expf(sc[jj] - m_new);
      ps[qi][sl + 16 * jj] = pv;
      psum += pv;
    }
#pragma unroll
    for (int off = 8; off > 0; off >>= 1) psum += __shfl_xor(psum, off);
    const float corr = (m == -INFINITY) ? 0.f : expf(m - m_new);
    l = l * corr + psum;
#pragma unroll
    for (int j = 0; j < ND; ++j) o[j] *= corr;
    m = m_new;
    __syncthreads();
    for (int kl = 0; kl < SUB; ++kl) {
      const float pv = ps[qi][kl];
#pragma unroll
      for (int j = 0; j < ND; ++j) {
        const int dim = sl + 16 * j;
        const uint32_t w = vs[kl][dim >> 1];
        o[j] += pv * ((dim & 1) ? bf_hi(w) : bf_lo(w));
      }
    }
  }

  // chunk partial: o [QB][HD], then m [QB], l [QB]
  constexpr int REC = QB * HD + 2 * QB;
  float* rec_base = p.part + ((size_t)(kvh * p.n_qblocks + z) * p.n_chunks) * REC;
  float* rec = rec_base + (size_t)c * REC;
#pragma unroll
  for (int j = 0; j < ND; ++j) rec[qi * HD + sl + 16 * j] = o[j];
  if (sl == 0) {
    rec[QB * HD + qi] = m;
    rec[QB * HD + QB + qi] = l;
  }
  __threadfence();
  __syncthreads();
  if (tid == 0) last_s = (atomicAdd(&p.counters[kvh * p.n_qblocks + z], 1) == n_act - 1);
  __syncthreads();
  if (!last_s) return;
  __threadfence();

  float M = -INFINITY;
  for (int cc = 0; cc < n_act; ++cc) M = fmaxf(M, rec_base[(size_t)cc * REC + QB * HD + qi]);
  float Lsum = 0.f;
  float acc[ND];
#pragma unroll
  for (int j = 0; j < ND; ++j) acc[j] = 0.f;
  for (int cc = 0; cc < n_act; ++cc) {
    const float* r = rec_base + (size_t)cc * REC;
    const float mc = r[QB * HD + qi];
    const float w = (mc == -INFINITY) ? 0.f : expf(mc - M);
    Lsum += r[QB * HD + QB + qi] * w;
#pragma unroll
    for (int j = 0; j < ND; ++j) acc[j] += r[qi * HD + sl + 16 * j] * w;
  }
  if (qh < n_qh) {
    const int row = qh / group, h = kvh * group + qh % group;
    const float inv = 1.0f / Lsum;
#pragma unroll
    for (int j = 0; j < ND; ++j) p.out[(size_t)row * p.ldo + h * HD + sl + 16 * j] = f2bf(acc[j] * inv);
  }
  if (tid == 0) p.counters[kvh * p.n_qblocks + z] = 0;
}

}  // namespace

size_t attn_part_floats(int head_dim) { return (size_t)kAttnQB * head_dim + 2 * kAttnQB; }

hipError_t launch_attention(int head_dim, const AttnArgs& a, hipStream_t st) {
  const dim3 grid(a.n_kv, a.n_chunks, a.n_qblocks), block(kBlock);
  if (head_dim == 64) {
    k_attn<64><<<grid, block, 0, st>>>(a);
  } else if (head_dim == 128) {
    k_attn<128><<<grid, block, 0, st>>>(a);
  } else {
    return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace pard
