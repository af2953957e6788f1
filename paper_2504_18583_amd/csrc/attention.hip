// Grouped-query causal attention of a short block of query rows against the
// bf16 KV cache (the draft pass with its mask rows, the verify pass, prefill
// chunks), on gfx950 MFMA.
//
// A workgroup serves one KV head, one block of 16*NQT (row, head-in-group)
// query pairs and one range of keys.  Per 32-key tile a wavefront computes
//   S^T[key][q] = K[key] . Q[q]          (v_mfma_f32_16x16x32_bf16, K rows as A,
//                                          Q as B, accumulated over head_dim)
//   O^T[dim][q] += V^T[dim][key] P^T[key][q]
// with an online softmax (running max m, sum l, fp32) in between.  The S^T
// accumulator of lane l holds keys 4g..4g+3 (and 16+4g..) for query l%16,
// g = l/16, which is exactly the B-operand fragment P^T needs once packed to
// bf16; the V cache stores each 32-key block transposed ([dim][key]) with those
// eight keys of group g contiguous, so V^T fragments are single 16-byte loads.
// K is cached row-major, so K fragments are 16-byte loads too.  Scores are
// causal by absolute position: key j is visible to the query at position
// pos0 + row iff j <= pos0 + row (mask rows of the draft pass are ordinary
// causal rows; Sec. 3.1 eq. 7 conditions candidate k on x_<n, m_0..m_{k-1}).
//
// The kAttnWaves wavefronts of a workgroup take its 32-key tiles round-robin
// and are merged in LDS in wave order.  With several key splits (long contexts) each workgroup writes
// (o, m, l) and k_attn_merge combines the splits in split order.  All
// reductions have a fixed order: results are deterministic and a query's
// result does not depend on the other rows of the pass.
#include "pard_internal.h"

namespace pard {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint32_t f2bf_bits(float f) {
  const uint32_t u = __float_as_uint(f);
  return (u + 0x7FFFu + ((u >> 16) & 1u)) >> 16;
}

template <int HD, int NQT>
__global__ __launch_bounds__(64 * kAttnWaves) void k_attn(const AttnArgs p) {
  constexpr int NWA = kAttnWaves;
  constexpr int QB = 16 * NQT;   // query pairs per block
  constexpr int KS = HD / 32;    // 32-dim steps of Q.K
  constexpr int DB = HD / 16;    // 16-dim blocks of the output
  __shared__ float mw[NWA][QB], lw[NWA][QB], fin_m[QB], fin_l[QB];
  __shared__ float ob[QB][HD + 1];

  const int kvh = blockIdx.x, z = blockIdx.y, sp = blockIdx.z;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int group = p.n_heads / p.n_kv;
  const FwdDesc d = *p.desc;
  const int L_end = d.pos0 + d.n_rows;
  const int n_qh = d.n_rows * group;
  if (z * QB >= n_qh) return;                      // uniform: the whole block leaves
  const int k_begin = sp * p.split_len;            // multiple of 32
  if (k_begin >= L_end) return;                    // uniform: split beyond the context
  const int k_end = min(L_end, k_begin + p.split_len);
  // wave w takes tiles w, w+NWA, ... of the split: the assignment does not
  // depend on where the pass ends, so tiles beyond a query's position add
  // exact zeros
  const int n_t = (k_end - k_begin + 31) / 32;
  const int n_my = (n_t - wave + NWA - 1) / NWA;

  const uint16_t* kbase = p.kc + (size_t)kvh * p.cap * HD;
  const uint16_t* vbase = p.vc + (size_t)kvh * p.cap * HD;
  const int g4 = lane >> 4, c16 = lane & 15;

  // Q fragments (B operand): query c16 of tile t, dims 32*ks + 8*g4 .. +7
  u32x4 qf[NQT][KS];
  int qpos[NQT];
#pragma unroll
  for (int t = 0; t < NQT; ++t) {
    const int qh = z * QB + t * 16 + c16;
    const bool ok = qh < n_qh;
    const int row = ok ? qh / group : 0;
    const int head = kvh * group + (ok ? qh % group : 0);
    qpos[t] = ok ? d.pos0 + row : -1;
    const uint16_t* qp = p.q + (size_t)row * p.ldq + head * HD + g4 * 8;
#pragma unroll
    for (int ks = 0; ks < KS; ++ks)
      qf[t][ks] = ok ? *reinterpret_cast<const u32x4*>(qp + ks * 32) : u32x4{0u, 0u, 0u, 0u};
  }

  float m[NQT], l[NQT];
  f32x4 o[DB][NQT];
#pragma unroll
  for (int t = 0; t < NQT; ++t) {
    m[t] = -INFINITY;
    l[t] = 0.f;
#pragma unroll
    for (int db = 0; db < DB; ++db) o[db][t] = f32x4{0.f, 0.f, 0.f, 0.f};
  }

  // two register stages of K and V fragments (tile i+1 loads while tile i computes)
  u32x4 kf0[2][KS], vf0[DB], kf1[2][KS], vf1[DB];
  auto load = [&](u32x4 (&kf)[2][KS], u32x4 (&vf)[DB], int it) {
    const int key0 = k_begin + (wave + NWA * min(it, n_my - 1)) * 32;   // in bounds: key0 + 31 < cap
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      const uint16_t* kp = kbase + (size_t)(key0 + kb * 16 + c16) * HD + g4 * 8;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) kf[kb][ks] = *reinterpret_cast<const u32x4*>(kp + ks * 32);
    }
    const uint16_t* vp = vbase + ((size_t)(key0 >> 5) * HD + c16) * 32 + g4 * 8;
#pragma unroll
    for (int db = 0; db < DB; ++db) vf[db] = *reinterpret_cast<const u32x4*>(vp + db * 16 * 32);
  };
  auto compute = [&](const u32x4 (&kf)[2][KS], const u32x4 (&vf)[DB], int it) {
    const int key0 = k_begin + (wave + NWA * it) * 32;
#pragma unroll
    for (int t = 0; t < NQT; ++t) {
      f32x4 s[2];
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        s[kb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
          s[kb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, kf[kb][ks]),
                                                          __builtin_bit_cast(bf16x8, qf[t][ks]), s[kb], 0, 0, 0);
      }
      float mx = -INFINITY;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int key = key0 + kb * 16 + g4 * 4 + i;
          const bool vis = key < k_end && key <= qpos[t];
          s[kb][i] = vis ? s[kb][i] * p.scale : -INFINITY;
          mx = fmaxf(mx, s[kb][i]);
        }
      mx = fmaxf(mx, __shfl_xor(mx, 16));
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      const float m_new = fmaxf(m[t], mx);
      const float corr = (m[t] == -INFINITY) ? 0.f : expf(m[t] - m_new);
      float pv[8];
      float rs = 0.f;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float e = (s[kb][i] == -INFINITY) ? 0.f : expf(s[kb][i] - m_new);
          pv[kb * 4 + i] = e;
          rs += e;
        }
      rs += __shfl_xor(rs, 16);
      rs += __shfl_xor(rs, 32);
      l[t] = l[t] * corr + rs;
      m[t] = m_new;
      u32x4 pf;
#pragma unroll
      for (int i = 0; i < 4; ++i) pf[i] = f2bf_bits(pv[2 * i]) | (f2bf_bits(pv[2 * i + 1]) << 16);
#pragma unroll
      for (int db = 0; db < DB; ++db) {
        o[db][t] *= corr;
        o[db][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, vf[db]),
                                                           __builtin_bit_cast(bf16x8, pf), o[db][t], 0, 0, 0);
      }
    }
  };
  if (n_my > 0) {
    int it = 0;
    load(kf0, vf0, it);
    while (true) {
      load(kf1, vf1, it + 1);
      __builtin_amdgcn_sched_barrier(0);
      compute(kf0, vf0, it);
      __builtin_amdgcn_sched_barrier(0);
      if (++it >= n_my) break;
      load(kf0, vf0, it + 1);
      __builtin_amdgcn_sched_barrier(0);
      compute(kf1, vf1, it);
      __builtin_amdgcn_sched_barrier(0);
      if (++it >= n_my) break;
    }
  }

  // ---- merge the wavefronts in wave order ----
  if (g4 == 0) {
#pragma unroll
    for (int t = 0; t < NQT; ++t) {
      mw[wave][t * 16 + c16] = m[t];
      lw[wave][t * 16 + c16] = l[t];
    }
  }
  __syncthreads();
  if (tid < QB) {
    float M = mw[0][tid];
    for (int w = 1; w < NWA; ++w) M = fmaxf(M, mw[w][tid]);
    float L = 0.f;
    for (int w = 0; w < NWA; ++w) L += (mw[w][tid] == -INFINITY) ? 0.f : lw[w][tid] * expf(mw[w][tid] - M);
    fin_m[tid] = M;
    fin_l[tid] = L;
  }
  __syncthreads();
  for (int w = 0; w < NWA; ++w) {
    if (wave == w) {
#pragma unroll
      for (int t = 0; t < NQT; ++t) {
        const int q = t * 16 + c16;
        const float f = (m[t] == -INFINITY) ? 0.f : expf(m[t] - fin_m[q]);
#pragma unroll
        for (int db = 0; db < DB; ++db)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            float& dst = ob[q][db * 16 + g4 * 4 + i];
            dst = (w == 0 ? 0.f : dst) + o[db][t][i] * f;
          }
      }
    }
    __syncthreads();
  }

  if (p.n_splits == 1) {
    for (int e = tid; e < QB * HD; e += 64 * NWA) {
      const int q = e / HD, dim = e % HD;
      const int qh = z * QB + q;
      if (qh < n_qh) {
        const int row = qh / group, head = kvh * group + qh % group;
        // same arithmetic as k_attn_merge with a single split
        p.out[act_index(row, head * HD + dim)] = (uint16_t)f2bf_bits(ob[q][dim] * (1.0f / fin_l[q]));
      }
    }
  } else {
    float* rec = p.part + ((size_t)(kvh * p.n_qblocks + z) * p.n_splits + sp) * (QB * HD + 2 * QB);
    for (int e = tid; e < QB * HD; e += 64 * NWA) rec[e] = ob[e / HD][e % HD];
    if (tid < QB) {
      rec[QB * HD + tid] = fin_m[tid];
      rec[QB * HD + QB + tid] = fin_l[tid];
    }
  }
}

// Combine the key splits of k_attn in split order.  Grid (kv head, query
// block, kMergeParts): per-query (max, sum) first, then each workgroup merges
// a slice of the (query, dim) outputs with 8 split loads in flight at a time.
constexpr int kMergeParts = 8;

template <int HD, int NQT>
__global__ __launch_bounds__(256) void k_attn_merge(const AttnArgs p) {
  constexpr int QB = 16 * NQT;
  constexpr int REC = QB * HD + 2 * QB;
  __shared__ float Ms[QB], Linv[QB];
  const int kvh = blockIdx.x, z = blockIdx.y, part = blockIdx.z, tid = threadIdx.x;
  const int group = p.n_heads / p.n_kv;
  const FwdDesc d = *p.desc;
  const int L_end = d.pos0 + d.n_rows;
  const int n_qh = d.n_rows * group;
  if (z * QB >= n_qh) return;                      // uniform
  const int n_act = min(p.n_splits, (L_end + p.split_len - 1) / p.split_len);
  const float* base = p.part + (size_t)(kvh * p.n_qblocks + z) * p.n_splits * REC;
  if (tid < QB) {
    float M = -INFINITY;
    for (int s = 0; s < n_act; ++s) M = fmaxf(M, base[(size_t)s * REC + QB * HD + tid]);
    float L = 0.f;
    for (int s = 0; s < n_act; ++s) {
      const float ms = base[(size_t)s * REC + QB * HD + tid];
      L += (ms == -INFINITY) ? 0.f : base[(size_t)s * REC + QB * HD + QB + tid] * expf(ms - M);
    }
    Ms[tid] = M;
    Linv[tid] = 1.0f / L;
  }
  __syncthreads();
  constexpr int PER = QB * HD / kMergeParts;
  for (int e = part * PER + tid; e < (part + 1) * PER; e += 256) {
    const int q = e / HD, dim = e % HD;
    const int qh = z * QB + q;
    if (qh >= n_qh) continue;
    const float M = Ms[q];
    float O = 0.f;
    for (int s0 = 0; s0 < n_act; s0 += 8) {
      float ov[8], mv[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int sx = min(s0 + u, n_act - 1);
        ov[u] = base[(size_t)sx * REC + e];
        mv[u] = base[(size_t)sx * REC + QB * HD + q];
      }
#pragma unroll
      for (int u = 0; u < 8; ++u)
        if (s0 + u < n_act && mv[u] != -INFINITY) O += ov[u] * expf(mv[u] - M);
    }
    const int row = qh / group, head = kvh * group + qh % group;
    p.out[act_index(row, head * HD + dim)] = (uint16_t)f2bf_bits(O * Linv[q]);
  }
}

template <int HD, int NQT>
hipError_t launch_hd_nqt(const AttnArgs& a, hipStream_t st) {
  k_attn<HD, NQT><<<dim3(a.n_kv, a.n_qblocks, a.n_splits), dim3(64 * kAttnWaves), 0, st>>>(a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || a.n_splits == 1) return e;
  k_attn_merge<HD, NQT><<<dim3(a.n_kv, a.n_qblocks, kMergeParts), dim3(256), 0, st>>>(a);
  return hipGetLastError();
}

template <int HD>
hipError_t launch_hd(const AttnArgs& a, hipStream_t st) {
  switch (a.nqt) {
    case 1: return launch_hd_nqt<HD, 1>(a, st);
    case 2: if constexpr (HD == 64) return launch_hd_nqt<HD, 2>(a, st); break;
  }
  return hipErrorInvalidValue;
}

}  // namespace

size_t attn_part_floats(int head_dim, int nqt) { return (size_t)16 * nqt * head_dim + 2 * 16 * nqt; }

hipError_t launch_attention(int head_dim, const AttnArgs& a, hipStream_t st) {
  if (a.split_len % 32 || a.split_len <= 0) return hipErrorInvalidValue;
  if (head_dim == 64) return launch_hd<64>(a, st);
  if (head_dim == 128) return launch_hd<128>(a, st);
  return hipErrorInvalidValue;
}

}  // namespace pard
