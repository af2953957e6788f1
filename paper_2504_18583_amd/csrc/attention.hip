// Grouped-query causal attention of a short block of query rows against the
// fp16 KV cache (the draft pass with its mask rows, the verify pass, prefill
// chunks), on gfx950 MFMA.  Q, K, V, the probabilities and the output are
// fp16 (10-bit mantissa: bf16 scores drift past the logit tolerance at 8B
// width).
//
// A workgroup serves one sequence of the pass, one KV head, one group of 16*NQ
// (row, head-in-group) query pairs -- for decode passes every pair of the KV
// head, so each key is read once per pass -- and one chunk of split_len keys
// (256 keys, two 32-key tiles per wavefront; decode passes over long contexts
// take longer chunks, multiples of 128 keys, so that their grid stays within
// one workgroup per CU).  Its four wavefronts take the
// chunk's tiles round-robin; per tile a wavefront computes
//   S^T[key][q] = K[key] . Q[q]          (v_mfma_f32_16x16x32_f16, K as A,
//                                          Q as B, accumulated over head_dim)
//   O^T[dim][q] += V^T[dim][key] P^T[key][q]
// with an online softmax (running max m, sum l, fp32, base 2) in between.  The
// S^T accumulator of lane l holds keys 4g..4g+3 (and 16+4g..) for query l%16,
// g = l/16, which is exactly the B-operand fragment P^T needs once packed to
// fp16; the V cache stores each 32-key block transposed ([dim][key]) with those
// eight keys of group g contiguous, and the K cache stores each 16-key block as
// ready A fragments, so every K or V fragment is one contiguous 1 KiB
// wavefront load.  Q fragments are staged once in LDS.
//
// Scores are causal by absolute position: key j is visible to the query at
// position pos0 + row iff j <= pos0 + row.  Mask rows of the draft pass are
// ordinary causal rows (Sec. 3.1, eq. 7: candidate k is conditioned on the
// prefix and the k-1 mask tokens before it).
//
// The wavefronts are merged in LDS in wave order.  With several chunks each
// workgroup writes (o, m, l) and a merge kernel combines them in a fixed order
// (k_attn_merge_few in chunk order for up to 16 chunks, k_attn_merge over lanes
// for more).
// All reductions have a fixed order, chunk boundaries sit at fixed multiples
// of split_len and a query's arithmetic does not depend on which other pairs
// share its workgroup: results are deterministic and a query's result does
// not depend on the other rows of the pass.  Chunks past a query's position
// contribute exact zeros.
#include "attn_tile.h"

namespace pard {
namespace {

using namespace attn;

// One workgroup per (KV head, query group, sequence x key chunk).
template <int HD, int NQ, int NW>
__global__ __launch_bounds__(64 * NW) void k_attn(const AttnArgs p) {
  __shared__ AttnLds<HD, NQ> sm;
  attn_tile<HD, NQ, NW, false>(p, blockIdx.x, blockIdx.y, blockIdx.z, FuseCtl{}, sm);
}

// Combine a few key chunks of k_attn (passes with many sequences or query
// groups and short contexts) in chunk order.  Grid (kv head, query group,
// sequence x kMergeParts): per-query (max, sum) first, then each thread merges
// 8 consecutive dims of one pair with the loads of 4 chunks in flight at a
// time.
constexpr int kMergeParts = 8;

template <int HD, int NQ>
__global__ __launch_bounds__(256) void k_attn_merge_few(const AttnArgs p) {
  constexpr int QP = 16 * NQ;
  constexpr int REC = QP * HD + 2 * QP;
  __shared__ float Ms[QP], Linv[QP];
  const int kvh = blockIdx.x, qg = blockIdx.y, tid = threadIdx.x;
  const int sj = blockIdx.z / kMergeParts, part = blockIdx.z % kMergeParts;
  const int group = p.n_heads / p.n_kv;
  if (sj >= p.desc->n_seq) return;                 // uniform
  const PassSeq d = p.desc->seq[sj];
  const int L_end = d.pos0 + d.n_rows;
  const int n_qh = d.n_rows * group;
  if (qg * QP >= n_qh) return;                     // uniform
  const int n_act = min(p.n_splits, (L_end + p.split_len - 1) / p.split_len);
  const float* base = p.part + ((size_t)(sj * p.n_kv + kvh) * p.n_qblocks + qg) * p.n_splits * REC;
  if (tid < QP) {
    // the (m, l) of up to 8 chunks are requested together
    float mv[8], lv[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const int sx = min(u, n_act - 1);
      mv[u] = base[(size_t)sx * REC + QP * HD + tid];
      lv[u] = base[(size_t)sx * REC + QP * HD + QP + tid];
    }
    float M = -INFINITY;
#pragma unroll
    for (int u = 0; u < 8; ++u)
      if (u < n_act) M = fmaxf(M, mv[u]);
    for (int s = 8; s < n_act; ++s) M = fmaxf(M, base[(size_t)s * REC + QP * HD + tid]);
    const float M_use = M == -INFINITY ? 0.f : M;
    float L = 0.f;
#pragma unroll
    for (int u = 0; u < 8; ++u)
      if (u < n_act) L += lv[u] * __builtin_amdgcn_exp2f(mv[u] - M_use);
    for (int s = 8; s < n_act; ++s)
      L += base[(size_t)s * REC + QP * HD + QP + tid] *
           __builtin_amdgcn_exp2f(base[(size_t)s * REC + QP * HD + tid] - M_use);
    Ms[tid] = M_use;
    Linv[tid] = 1.0f / L;
  }
  __syncthreads();
  constexpr int NV = QP * HD / 8;                  // 8-dim vectors of the group
  constexpr int PER = (NV + kMergeParts - 1) / kMergeParts;
  for (int e = part * PER + tid; e < min(NV, (part + 1) * PER); e += 256) {
    const int q = e / (HD / 8), d0 = (e % (HD / 8)) * 8;
    const int qh = qg * QP + q;
    if (qh >= n_qh) continue;
    const float M = Ms[q];
    f32x4 a = f32x4{0.f, 0.f, 0.f, 0.f}, b = a;
    for (int s0 = 0; s0 < n_act; s0 += 4) {
      f32x4 va[4], vb[4];
      float mv[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int sx = min(s0 + u, n_act - 1);
        const float* r = base + (size_t)sx * REC;
        va[u] = *reinterpret_cast<const f32x4*>(r + q * HD + d0);
        vb[u] = *reinterpret_cast<const f32x4*>(r + q * HD + d0 + 4);
        mv[u] = r[QP * HD + q];
      }
#pragma unroll
      for (int u = 0; u < 4; ++u)
        if (s0 + u < n_act) {
          const float sc = __builtin_amdgcn_exp2f(mv[u] - M);
          a += va[u] * sc;
          b += vb[u] * sc;
        }
    }
    const int row = qh / group, head = kvh * group + qh % group;
    store_f16x8(p.out + act_index(d.row0 + row, head * HD + d0, p.act_rows), a * Linv[q], b * Linv[q]);
  }
}

// Combine many key chunks of k_attn (long contexts).  One workgroup per (KV
// head, query group, sequence, 16 output vectors of 8 dims), so that the
// chunks spread over many workgroups and lanes.  (With few chunks its many
// small workgroups cost more than they save: batch-32 step 15.8 -> 16.7 ms.)  The chunks are dealt round-robin over
// lanes, every lane folds its chunks in chunk order with all of its loads in
// flight together, and lanes are combined in a fixed tree order: the result
// is deterministic and no lane waits on more than one round of loads for
// contexts up to 16 x kAttnChunk x 8 keys.
//   (1) per query pair of the workgroup: the running (max, sum) of its chunks'
//       (m, l) over lanes, then the combination over lanes (wavefront
//       shuffles, then the wavefronts in order);
//   (2) per output vector: 16 lanes add o_chunk * 2^(m_chunk - M), then a
//       shuffle tree; lane 0 stores o / L.
constexpr int kMergeFewChunks = 16;   // up to this many chunks: k_attn_merge_few
constexpr int kMergeVecs = 16;     // 8-dim output vectors per workgroup
constexpr int kMergeLanes = 16;    // lanes (chunk subsets) per vector

// (m, l) of two partial softmax sums combined: the larger max is kept and the
// other sum rescaled (an empty part has m = -inf, l = 0).
__device__ __forceinline__ void ml_combine(float& m, float& l, float m2, float l2) {
  const float M = fmaxf(m, m2);
  const float Mu = M == -INFINITY ? 0.f : M;
  l = l * __builtin_amdgcn_exp2f(m - Mu) + l2 * __builtin_amdgcn_exp2f(m2 - Mu);
  m = M;
}

template <int HD, int NQ>
constexpr int merge_parts() { return (16 * NQ * HD / 8 + kMergeVecs - 1) / kMergeVecs; }

template <int HD, int NQ>
__global__ __launch_bounds__(256) void k_attn_merge(const AttnArgs p) {
  constexpr int QP = 16 * NQ;
  constexpr int REC = QP * HD + 2 * QP;
  constexpr int VPQ = HD / 8;                      // output vectors per query pair
  constexpr int NPAIR = (kMergeVecs + VPQ - 1) / VPQ;   // pairs a workgroup touches (1 or 2)
  constexpr int TPP = 256 / NPAIR;                 // step (1) lanes per pair: whole wavefronts
  constexpr int WPP = TPP / 64;
  constexpr int PARTS = merge_parts<HD, NQ>();
  static_assert(VPQ % kMergeVecs == 0 || kMergeVecs % VPQ == 0, "vectors of a workgroup cover whole pairs");
  __shared__ float wm_s[4], wl_s[4], M_s[NPAIR], Linv_s[NPAIR];
  const int kvh = blockIdx.x, qg = blockIdx.y, tid = threadIdx.x, lane = tid & 63;
  const int sj = blockIdx.z / PARTS, part = blockIdx.z % PARTS;
  const int group = p.n_heads / p.n_kv;
  if (sj >= p.desc->n_seq) return;                 // uniform
  const PassSeq d = p.desc->seq[sj];
  const int L_end = d.pos0 + d.n_rows;
  const int n_qh = d.n_rows * group;
  if (qg * QP >= n_qh) return;                     // uniform
  const int n_act = min(p.n_splits, (L_end + p.split_len - 1) / p.split_len);
  const float* base = p.part + ((size_t)(sj * p.n_kv + kvh) * p.n_qblocks + qg) * p.n_splits * REC;
  const int v0 = part * kMergeVecs;                // first output vector of the workgroup
  const int q0 = v0 / VPQ;                         // its first pair

  // (1) (max, sum) of pair q0 + tid / TPP over its chunks
  {
    const int pi = tid / TPP, ln = tid % TPP;
    const int q = min(q0 + pi, QP - 1);
    float m = -INFINITY, l = 0.f;
    for (int s0 = ln; s0 < n_act; s0 += 4 * TPP) {
      float mv[4], lv[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int sx = min(s0 + u * TPP, n_act - 1);
        mv[u] = base[(size_t)sx * REC + QP * HD + q];
        lv[u] = base[(size_t)sx * REC + QP * HD + QP + q];
      }
#pragma unroll
      for (int u = 0; u < 4; ++u)
        if (s0 + u * TPP < n_act) ml_combine(m, l, mv[u], lv[u]);
    }
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const float m2 = __shfl_xor(m, off), l2 = __shfl_xor(l, off);
      // lower lane first: both lanes hold the same combination
      if (lane & off) { float mm = m2, ll = l2; ml_combine(mm, ll, m, l); m = mm; l = ll; }
      else ml_combine(m, l, m2, l2);
    }
    if (lane == 0) { wm_s[tid >> 6] = m; wl_s[tid >> 6] = l; }
    __syncthreads();
    if (tid < NPAIR) {
      float M = wm_s[tid * WPP], L = wl_s[tid * WPP];
      for (int w = 1; w < WPP; ++w) ml_combine(M, L, wm_s[tid * WPP + w], wl_s[tid * WPP + w]);
      M_s[tid] = M == -INFINITY ? 0.f : M;
      Linv_s[tid] = 1.0f / L;
    }
    __syncthreads();
  }

  // (2) output vector v0 + tid / kMergeLanes
  const int v = v0 + tid / kMergeLanes, ln = tid % kMergeLanes;
  const int q = v / VPQ, d0 = (v % VPQ) * 8;
  const int qc = min(q, QP - 1);
  const float M = M_s[min(qc - q0, NPAIR - 1)];
  f32x4 a = f32x4{0.f, 0.f, 0.f, 0.f}, b = a;
  for (int s0 = ln; s0 < n_act; s0 += 4 * kMergeLanes) {
    f32x4 va[4], vb[4];
    float mv[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      const int sx = min(s0 + u * kMergeLanes, n_act - 1);
      const float* r = base + (size_t)sx * REC;
      va[u] = *reinterpret_cast<const f32x4*>(r + qc * HD + d0);
      vb[u] = *reinterpret_cast<const f32x4*>(r + qc * HD + d0 + 4);
      mv[u] = r[QP * HD + qc];
    }
#pragma unroll
    for (int u = 0; u < 4; ++u)
      if (s0 + u * kMergeLanes < n_act) {
        const float sc = __builtin_amdgcn_exp2f(mv[u] - M);
        a += va[u] * sc;
        b += vb[u] * sc;
      }
  }
#pragma unroll
  for (int off = 1; off < kMergeLanes; off <<= 1) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      // lower lane's value first, so both lanes of a pair hold the same sum
      const float a2 = __shfl_xor(a[i], off), b2 = __shfl_xor(b[i], off);
      a[i] = (lane & off) ? a2 + a[i] : a[i] + a2;
      b[i] = (lane & off) ? b2 + b[i] : b[i] + b2;
    }
  }
  const int qh = qg * QP + q;
  if (ln == 0 && q < QP && qh < n_qh) {
    const float li = Linv_s[min(qc - q0, NPAIR - 1)];
    const int row = qh / group, head = kvh * group + qh % group;
    store_f16x8(p.out + act_index(d.row0 + row, head * HD + d0, p.act_rows), a * li, b * li);
  }
}

template <int HD, int NQ>
hipError_t launch_hd_nq(const AttnArgs& a, hipStream_t st) {
  if (a.wide) {                      // one chunk, 8 waves: no merge kernel
    k_attn<HD, NQ, 2 * kAttnWaves><<<dim3(a.n_kv, a.n_qblocks, a.n_seq), dim3(128 * kAttnWaves), 0, st>>>(a);
    return hipGetLastError();
  }
  k_attn<HD, NQ, kAttnWaves><<<dim3(a.n_kv, a.n_qblocks, a.n_seq * a.n_splits), dim3(64 * kAttnWaves), 0, st>>>(a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || a.n_splits == 1) return e;
  if (a.n_splits <= kMergeFewChunks)
    k_attn_merge_few<HD, NQ><<<dim3(a.n_kv, a.n_qblocks, a.n_seq * kMergeParts), dim3(256), 0, st>>>(a);
  else
    k_attn_merge<HD, NQ><<<dim3(a.n_kv, a.n_qblocks, a.n_seq * merge_parts<HD, NQ>()), dim3(256), 0, st>>>(a);
  return hipGetLastError();
}

template <int HD>
hipError_t launch_hd(const AttnArgs& a, hipStream_t st) {
  switch (a.nqt) {
    case 1: return launch_hd_nq<HD, 1>(a, st);
    case 2: return launch_hd_nq<HD, 2>(a, st);
    case 3: return launch_hd_nq<HD, 3>(a, st);
    case 4: if constexpr (HD == 64) return launch_hd_nq<HD, 4>(a, st); break;
  }
  return hipErrorInvalidValue;
}

}  // namespace

int attn_max_q_tiles(int head_dim) { return head_dim == 128 ? 3 : 4; }

size_t attn_part_floats(int head_dim, int nqt) { return (size_t)16 * nqt * head_dim + 2 * 16 * nqt; }

hipError_t launch_attention(int head_dim, const AttnArgs& a, hipStream_t st) {
  if (a.split_len % 128 || a.split_len <= 0) return hipErrorInvalidValue;
  if (a.nqt < 1 || a.nqt > attn_max_q_tiles(head_dim)) return hipErrorInvalidValue;
  if (a.n_seq < 1 || a.n_seq > kMaxPassSeqs || (size_t)a.n_seq * a.n_splits > 65535) return hipErrorInvalidValue;
  if (a.wide && a.n_splits != 1) return hipErrorInvalidValue;
  if (head_dim == 64) return launch_hd<64>(a, st);
  if (head_dim == 128) return launch_hd<128>(a, st);
  return hipErrorInvalidValue;
}

}  // namespace pard
