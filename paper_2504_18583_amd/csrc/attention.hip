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
#include "pard_internal.h"

namespace pard {
namespace {

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

typedef float f32x2 __attribute__((ext_vector_type(2)));

typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));

// two floats to packed fp16, round to nearest even (v_cvt_pk_f16_f32)
__device__ __forceinline__ uint32_t pack_f16x2(float a, float b) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{a, b}, f16x2));
}

// 8 consecutive fp16 outputs as one 16-byte store
__device__ __forceinline__ void store_f16x8(uint16_t* dst, f32x4 a, f32x4 b) {
  *reinterpret_cast<u32x4*>(dst) = u32x4{pack_f16x2(a[0], a[1]), pack_f16x2(a[2], a[3]),
                                         pack_f16x2(b[0], b[1]), pack_f16x2(b[2], b[3])};
}

constexpr float kLog2e = 1.4426950408889634f;

// Reductions across lanes l and l^16 / l^32 with the gfx950 lane-swap
// instructions (VALU, no LDS round trip).  Both lanes of a pair combine the
// same two operands in the same order.
__device__ __forceinline__ f32x2 swap16(float x) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return f32x2{__uint_as_float(r[0]), __uint_as_float(r[1])};
}
__device__ __forceinline__ f32x2 swap32(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return f32x2{__uint_as_float(r[0]), __uint_as_float(r[1])};
}
__device__ __forceinline__ float max4g(float x) {    // max over the 4 lane groups (l, l^16, l^32, l^48)
  f32x2 r = swap16(x);
  x = fmaxf(r[0], r[1]);
  r = swap32(x);
  return fmaxf(r[0], r[1]);
}
__device__ __forceinline__ float sum4g(float x) {
  f32x2 r = swap16(x);
  x = r[0] + r[1];
  r = swap32(x);
  return r[0] + r[1];
}

// NW wavefronts per workgroup: kAttnWaves (4) for chunked passes, 2 * kAttnWaves
// (8) for short contexts covered by one chunk -- there waves 4..7 first fold
// their (m, l, o) into waves 0..3 through LDS (wave w + 4 into wave w), so
// that the wave merge below and its LDS stay those of 4 waves.
template <int HD, int NQ, int NW>
__global__ __launch_bounds__(64 * NW) void k_attn(const AttnArgs p) {
  constexpr int NWA = NW;
  constexpr int MW = kAttnWaves;     // waves in the final LDS merge
  constexpr int QP = 16 * NQ;        // query pairs per workgroup
  constexpr int KS = HD / 32;        // 32-dim steps of Q.K
  constexpr int DB = HD / 16;        // 16-dim blocks of the output
  constexpr int OS = HD + 4;         // row stride of the per-wave output tiles in LDS
  constexpr int REC = QP * HD + 2 * QP;   // floats of one chunk record: o [QP][HD], m [QP], l [QP]
  __shared__ u32x4 q_lds[NQ * KS * 64];   // Q fragments in B-operand lane order
  __shared__ __attribute__((aligned(16))) float o_lds[MW][QP][OS];
  __shared__ float m_lds[MW][QP], l_lds[MW][QP], sc_lds[MW][QP], linv_lds[QP];

  const int kvh = blockIdx.x, qg = blockIdx.y;
  const int sj = blockIdx.z / p.n_splits, ch = blockIdx.z % p.n_splits;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int group = p.n_heads / p.n_kv;
  if (sj >= p.desc->n_seq) return;                 // uniform: the whole block leaves
  const PassSeq d = p.desc->seq[sj];
  const int L_end = d.pos0 + d.n_rows;
  const int n_qh = d.n_rows * group;
  if (qg * QP >= n_qh) return;                     // uniform
  const int k_begin = ch * p.split_len;            // multiple of 128
  if (k_begin >= L_end) return;                    // uniform: chunk beyond the context
  const int k_end = min(L_end, k_begin + p.split_len);
  // wave w takes tiles w, w+NWA, ... of the chunk: the assignment does not
  // depend on where the pass ends, so tiles beyond a query's position add
  // exact zeros
  const int n_t = (k_end - k_begin + 31) / 32;
  const int n_my = (n_t - wave + NWA - 1) / NWA;

  const size_t cache = (size_t)d.slot * p.kv_seq_stride + (size_t)kvh * p.cap * HD;
  const uint16_t* kbase = p.kc + cache;
  const uint16_t* vbase = p.vc + cache;
  const int g4 = lane >> 4, c16 = lane & 15;

  // K and V fragments of two tiles (a pair of tiles shares one softmax max)
  u32x4 kf[2][2][KS], vf[2][DB];
  // a wave with no tile of its own (n_my = 0) reads the chunk's first tile
  // and never uses it; in bounds: key0 + 31 < cap
  auto tile_key = [&](int it) { return k_begin + (n_my > 0 ? wave + NWA * min(it, n_my - 1) : 0) * 32; };
  auto load_k = [&](int tt, int it) {
    const int key0 = tile_key(it);
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      const uint16_t* kp = kbase + ((size_t)((key0 >> 4) + kb) * KS * 64 + lane) * 8;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) kf[tt][kb][ks] = *reinterpret_cast<const u32x4*>(kp + ks * 64 * 8);
    }
  };
  auto load_v = [&](int tt, int it) {
    const int key0 = tile_key(it);
    const uint16_t* vp = vbase + ((size_t)(key0 >> 5) * HD + c16) * 32 + g4 * 8;
#pragma unroll
    for (int db = 0; db < DB; ++db) vf[tt][db] = *reinterpret_cast<const u32x4*>(vp + db * 16 * 32);
  };
  auto load = [&](int tt, int it) {
    load_k(tt, it);
    load_v(tt, it);
  };

  // stage the Q fragments: entry (t, ks, l) = pair t*16 + l%16, dims ks*32 + 8*(l/16) .. +7.
  // Their loads go out before the K/V loads (returns are in order per wavefront).
  // All of these loads are unconditional (entries past the group re-read a
  // valid one and are zeroed; a wave without tiles reads the chunk's first):
  // a branch around any of them would make the wait for Q below also wait for
  // every K/V load in flight.
  constexpr int QE = (NQ * KS * 64 + 64 * NWA - 1) / (64 * NWA);   // entries per thread
  u32x4 qv[QE];
#pragma unroll
  for (int j = 0; j < QE; ++j) {
    const int e = tid + j * 64 * NWA;
    const int ec = min(e, NQ * KS * 64 - 1);
    const int t = ec / (KS * 64), ks = (ec / 64) % KS, l = ec & 63;
    const int qh = qg * QP + t * 16 + (l & 15);
    const int qhc = min(qh, n_qh - 1);
    const int row = qhc / group, head = kvh * group + qhc % group;
    const u32x4 v = *reinterpret_cast<const u32x4*>(p.q + (size_t)(d.row0 + row) * p.ldq + head * HD + ks * 32 +
                                                    (l >> 4) * 8);
    qv[j] = (e < NQ * KS * 64 && qh < n_qh) ? v : u32x4{0u, 0u, 0u, 0u};
  }
  __builtin_amdgcn_sched_barrier(0);                // Q's loads, then both tiles' K, then V
  load_k(0, 0);
  load_k(1, 1);
  __builtin_amdgcn_sched_barrier(0);
  load_v(0, 0);
  load_v(1, 1);
  __builtin_amdgcn_sched_barrier(0);
#pragma unroll
  for (int j = 0; j < QE; ++j) {
    const int e = tid + j * 64 * NWA;
    if (e < NQ * KS * 64) q_lds[e] = qv[j];
  }
  int qpos[NQ];
#pragma unroll
  for (int t = 0; t < NQ; ++t) {
    const int qh = qg * QP + t * 16 + c16;
    qpos[t] = qh < n_qh ? d.pos0 + qh / group : -1;
  }
  __syncthreads();

  float m[NQ], l[NQ];
  f32x4 o[NQ][DB];
#pragma unroll
  for (int t = 0; t < NQ; ++t) {
    m[t] = -INFINITY;
    l[t] = 0.f;
#pragma unroll
    for (int db = 0; db < DB; ++db) o[t][db] = f32x4{0.f, 0.f, 0.f, 0.f};
  }
  const float scale2 = p.scale * kLog2e;   // scores in base 2

  for (int it0 = 0; it0 < n_my; it0 += 2) {
    const int nt = min(2, n_my - it0);     // tiles in this pair (uniform)
    if (it0 > 0) {
      load(0, it0);
      if (nt > 1) load(1, it0 + 1);
    }
    // scores of every query tile first, then the softmax of all of them, so
    // the dependent steps of different query tiles overlap
    f32x4 s[NQ][2][2];
#pragma unroll
    for (int t = 0; t < NQ; ++t)
#pragma unroll
      for (int tt = 0; tt < 2; ++tt)
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) {
          s[t][tt][kb] = f32x4{0.f, 0.f, 0.f, 0.f};
          if (tt == 0 || nt > 1) {             // uniform: the second tile may be absent
#pragma unroll
            for (int ks = 0; ks < KS; ++ks)
              s[t][tt][kb] = __builtin_amdgcn_mfma_f32_16x16x32_f16(
                  __builtin_bit_cast(f16x8, kf[tt][kb][ks]), __builtin_bit_cast(f16x8, q_lds[(t * KS + ks) * 64 + lane]),
                  s[t][tt][kb], 0, 0, 0);
          }
        }
    // causal / range mask; only tiles that reach past the context end or the
    // first query's position need it
#pragma unroll
    for (int tt = 0; tt < 2; ++tt) {
      const int key0 = k_begin + (wave + NWA * (it0 + tt)) * 32;
      if (tt >= nt || key0 + 31 >= k_end || key0 + 31 > d.pos0) {
#pragma unroll
        for (int t = 0; t < NQ; ++t)
#pragma unroll
          for (int kb = 0; kb < 2; ++kb)
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const int key = key0 + kb * 16 + g4 * 4 + i;
              if (tt >= nt || key >= k_end || key > qpos[t]) s[t][tt][kb][i] = -INFINITY;
            }
      }
    }
    float mx[NQ];
#pragma unroll
    for (int t = 0; t < NQ; ++t) {
      mx[t] = -INFINITY;
#pragma unroll
      for (int tt = 0; tt < 2; ++tt)
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int i = 0; i < 4; ++i) mx[t] = fmaxf(mx[t], s[t][tt][kb][i]);
    }
#pragma unroll
    for (int t = 0; t < NQ; ++t) mx[t] = max4g(mx[t]);
    float corr[NQ], rs[NQ];
    u32x4 pf[NQ][2];
#pragma unroll
    for (int t = 0; t < NQ; ++t) {
      const float m_new = fmaxf(m[t], mx[t] * scale2);
      const float m_use = m_new == -INFINITY ? 0.f : m_new;   // keeps 2^(-inf - m) = 0 well defined
      corr[t] = __builtin_amdgcn_exp2f(m[t] - m_use);
      m[t] = m_new;
      rs[t] = 0.f;
#pragma unroll
      for (int tt = 0; tt < 2; ++tt) {
        float pv[8];
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            pv[kb * 4 + i] = __builtin_amdgcn_exp2f(fmaf(s[t][tt][kb][i], scale2, -m_use));
            rs[t] += pv[kb * 4 + i];
          }
#pragma unroll
        for (int i = 0; i < 4; ++i) pf[t][tt][i] = pack_f16x2(pv[2 * i], pv[2 * i + 1]);
      }
    }
#pragma unroll
    for (int t = 0; t < NQ; ++t) l[t] = l[t] * corr[t] + sum4g(rs[t]);
#pragma unroll
    for (int t = 0; t < NQ; ++t) {
      if (it0 > 0) {                       // uniform; o is still zero for the first pair
#pragma unroll
        for (int db = 0; db < DB; ++db) o[t][db] *= corr[t];
      }
#pragma unroll
      for (int tt = 0; tt < 2; ++tt)
        if (tt == 0 || nt > 1) {
#pragma unroll
          for (int db = 0; db < DB; ++db)
            o[t][db] = __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, vf[tt][db]),
                                                               __builtin_bit_cast(f16x8, pf[t][tt]), o[t][db], 0, 0, 0);
        }
    }
  }

  // ---- merge the wavefronts in wave order ----
  // lane (c16, g4) holds dims db*16 + 4*g4 .. +3 of pair t*16 + c16
  auto publish = [&](int slot) {
    if (g4 == 0) {
#pragma unroll
      for (int t = 0; t < NQ; ++t) {
        m_lds[slot][t * 16 + c16] = m[t];
        l_lds[slot][t * 16 + c16] = l[t];
      }
    }
#pragma unroll
    for (int t = 0; t < NQ; ++t)
#pragma unroll
      for (int db = 0; db < DB; ++db)
        *reinterpret_cast<f32x4*>(&o_lds[slot][t * 16 + c16][db * 16 + g4 * 4]) = o[t][db];
  };
  if constexpr (NW > MW) {
    static_assert(NW == 2 * MW, "the fold pairs wave w + MW with wave w");
    if (wave >= MW) publish(wave - MW);
    __syncthreads();
    if (wave < MW) {
#pragma unroll
      for (int t = 0; t < NQ; ++t) {
        const float mb = m_lds[wave][t * 16 + c16], lb = l_lds[wave][t * 16 + c16];
        const float mn = fmaxf(m[t], mb);
        const float mu = mn == -INFINITY ? 0.f : mn;
        const float sa = __builtin_amdgcn_exp2f(m[t] - mu), sb = __builtin_amdgcn_exp2f(mb - mu);
        l[t] = l[t] * sa + lb * sb;
        m[t] = mn;
#pragma unroll
        for (int db = 0; db < DB; ++db)
          o[t][db] = o[t][db] * sa + *reinterpret_cast<const f32x4*>(&o_lds[wave][t * 16 + c16][db * 16 + g4 * 4]) * sb;
      }
    }
    __syncthreads();
  }
  if (wave < MW) publish(wave);
  __syncthreads();
  float* rec = p.part + (((size_t)(sj * p.n_kv + kvh) * p.n_qblocks + qg) * p.n_splits + ch) * REC;   // this chunk's record
  if (tid < QP) {
    float M = m_lds[0][tid];
    for (int w = 1; w < MW; ++w) M = fmaxf(M, m_lds[w][tid]);
    const float M_use = M == -INFINITY ? 0.f : M;
    float L = 0.f;
    for (int w = 0; w < MW; ++w) {
      const float sc = __builtin_amdgcn_exp2f(m_lds[w][tid] - M_use);
      sc_lds[w][tid] = sc;
      L += l_lds[w][tid] * sc;
    }
    if (p.n_splits == 1) {
      linv_lds[tid] = 1.0f / L;            // same arithmetic as the chunk merge with one chunk
    } else {
      rec[QP * HD + tid] = M;
      rec[QP * HD + QP + tid] = L;
    }
  }
  __syncthreads();
  // each thread finishes 8 consecutive dims of one pair: one 16-byte fp16
  // store (or two 16-byte fp32 stores of the chunk record)
  for (int e = tid; e < QP * HD / 8; e += 64 * NWA) {
    const int q = e / (HD / 8), d0 = (e % (HD / 8)) * 8;
    f32x4 a = f32x4{0.f, 0.f, 0.f, 0.f}, b = a;
#pragma unroll
    for (int w = 0; w < MW; ++w) {
      const float sc = sc_lds[w][q];
      a += *reinterpret_cast<const f32x4*>(&o_lds[w][q][d0]) * sc;
      b += *reinterpret_cast<const f32x4*>(&o_lds[w][q][d0 + 4]) * sc;
    }
    if (p.n_splits == 1) {
      const int qh = qg * QP + q;
      if (qh < n_qh) {
        const int row = qh / group, head = kvh * group + qh % group;
        store_f16x8(p.out + act_index(d.row0 + row, head * HD + d0, p.act_rows), a * linv_lds[q], b * linv_lds[q]);
      }
    } else {
      *reinterpret_cast<f32x4*>(rec + q * HD + d0) = a;
      *reinterpret_cast<f32x4*>(rec + q * HD + d0 + 4) = b;
    }
  }
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
