// Attention tile of one workgroup: (sequence, KV head, query group, key
// chunk) -- shared by the attention kernels and the QKV GEMM launch that
// carries decode attention (see k_attn and k_qkv_attn).
//
// Grouped-query causal attention of a short block of query rows against the
// fp16 KV cache; the layout and algorithm are described in attention.hip.
#pragma once

#include "pard_internal.h"

namespace pard {
namespace attn {

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


constexpr int kRsrcWord3 = 0x00020000;     // buffer descriptor word 3 for gfx9-family raw buffers
constexpr int kCachePolicyDevice = 16;     // sc1: device scope, coherent across XCDs
constexpr int kFuseSpinLimit = 1 << 20;    // polls before a fused wait gives up (and flags an error)

// Wait until the LANES (at most kFuseLanes) counters at `lanes`, kFuseStride
// ints apart, add up to n: many arrivals are spread over the counters (one
// per XCD when workgroups are dealt round-robin over the XCDs) so that their
// device-scope atomics do not all meet on one address; few arrivals awaited
// by many pollers go to every counter and each poller reads one (measured:
// one shared counter for all pollers is slower, as are arrivals on every
// counter for the QKV workgroups).
// Wavefront 0 polls (lane j reads counter j, the lanes add them up with DPP
// moves); the other wavefronts wait at the workgroup barrier with their loads
// still in flight.  One poll at a time: keeping four in flight per poller
// measured slower (their loads delay the arrivals' atomics on the same lines).
// Every wavefront of the workgroup must call this.  The spin is bounded: past
// kFuseSpinLimit polls the wait sets *err and returns (the results are then
// invalid and the host reports an error), so no wavefront waits forever.
template <int LANES>
__device__ __forceinline__ void fuse_wait_on(const int* lanes, const int n, int* err) {
  if (threadIdx.x < 64) {
    const int lane = threadIdx.x;
    // every lane loads (lanes past the counters re-read the last one and are
    // not counted): no branch around the load
    const int* addr = lanes + min(lane, LANES - 1) * kFuseStride;
    for (int spins = 0;; ++spins) {
      int v = __hip_atomic_load(addr, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      v = lane < LANES ? v : 0;
      v += __builtin_amdgcn_mov_dpp(v, 0xB1, 0xF, 0xF, false);    // quad_perm 1 0 3 2
      v += __builtin_amdgcn_mov_dpp(v, 0x4E, 0xF, 0xF, false);    // quad_perm 2 3 0 1
      v += __builtin_amdgcn_mov_dpp(v, 0x141, 0xF, 0xF, false);   // half-row mirror: the other quad
      if (__builtin_amdgcn_readfirstlane(v) >= n) break;
      if (spins >= kFuseSpinLimit) {
        if (lane == 0) __hip_atomic_store(err, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        break;
      }
      __builtin_amdgcn_s_sleep(4);
    }
  }
  __builtin_amdgcn_s_barrier();
}

// Wait for every QKV workgroup of the launch.
__device__ __forceinline__ void fuse_wait(const FuseCtl& f) { fuse_wait_on<kFuseLanes>(f.counters, f.n_prod, f.err); }

// The attention tile's LDS arrays: Q fragments in B-operand lane order, and the
// wavefronts' output tiles and softmax statistics for the final merge.  The
// kernel declares them (static LDS, so the compiler keeps them apart from its
// dynamic LDS), and a fused launch reuses them once the tile is done.
template <int HD, int NQ>
struct AttnLds {
  u32x4 q[NQ * (HD / 32) * 64];
  float o[kAttnWaves][16 * NQ][HD + 4];
  float m[kAttnWaves][16 * NQ], l[kAttnWaves][16 * NQ], sc[kAttnWaves][16 * NQ], linv[16 * NQ];
};

template <int HD, int NQ, int NW, bool FUSED>
__device__ __forceinline__ void attn_tile(const AttnArgs& p, const int kvh, const int qg, const unsigned zz,
                                          const FuseCtl& fc, AttnLds<HD, NQ>& sm) {
  constexpr int NWA = NW;
  constexpr int MW = kAttnWaves;     // waves in the final LDS merge
  constexpr int QP = 16 * NQ;        // query pairs per workgroup
  constexpr int KS = HD / 32;        // 32-dim steps of Q.K
  constexpr int DB = HD / 16;        // 16-dim blocks of the output
  constexpr int OS = HD + 4;         // row stride of the per-wave output tiles in LDS
  constexpr int REC = QP * HD + 2 * QP;   // floats of one chunk record: o [QP][HD], m [QP], l [QP]
  static_assert(MW == kAttnWaves && OS == HD + 4 && QP == 16 * NQ, "AttnLds holds the tile's arrays");
  auto& q_lds = sm.q;
  auto& o_lds = sm.o;
  auto& m_lds = sm.m;
  auto& l_lds = sm.l;
  auto& sc_lds = sm.sc;
  auto& linv_lds = sm.linv;

  const int sj = zz / p.n_splits, ch = zz % p.n_splits;
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
  // Fused with the QKV GEMM (FUSED): a tile that holds a key at or past the
  // pass's first position was written in this launch by another workgroup,
  // so it is read with device-scope loads (coherent across XCDs) after the
  // wait; tiles wholly before it were written by earlier launches.
  auto fresh = [&](int it) { return FUSED && tile_key(it) + 31 >= d.pos0; };
  const __amdgpu_buffer_rsrc_t krs = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(kbase), 0,
                                                                        p.cap * HD * 2, kRsrcWord3);
  const __amdgpu_buffer_rsrc_t vrs = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(vbase), 0,
                                                                        p.cap * HD * 2, kRsrcWord3);
  auto load_k = [&](int tt, int it) {
    const int key0 = tile_key(it);
    if (fresh(it)) {                               // uniform
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        const int off = (((key0 >> 4) + kb) * KS * 64 + lane) * 8;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
          kf[tt][kb][ks] = __builtin_amdgcn_raw_buffer_load_b128(krs, (off + ks * 64 * 8) * 2, 0, kCachePolicyDevice);
      }
      return;
    }
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      const uint16_t* kp = kbase + ((size_t)((key0 >> 4) + kb) * KS * 64 + lane) * 8;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) kf[tt][kb][ks] = *reinterpret_cast<const u32x4*>(kp + ks * 64 * 8);
    }
  };
  auto load_v = [&](int tt, int it) {
    const int key0 = tile_key(it);
    if (fresh(it)) {
      const int off = ((key0 >> 5) * HD + c16) * 32 + g4 * 8;
#pragma unroll
      for (int db = 0; db < DB; ++db)
        vf[tt][db] = __builtin_amdgcn_raw_buffer_load_b128(vrs, (off + db * 16 * 32) * 2, 0, kCachePolicyDevice);
      return;
    }
    const uint16_t* vp = vbase + ((size_t)(key0 >> 5) * HD + c16) * 32 + g4 * 8;
#pragma unroll
    for (int db = 0; db < DB; ++db) vf[tt][db] = *reinterpret_cast<const u32x4*>(vp + db * 16 * 32);
  };
  auto load = [&](int tt, int it) {
    load_k(tt, it);
    load_v(tt, it);
  };
  // FUSED: the first pair of tiles, when both precede the pass, is requested
  // before waiting for the QKV workgroups
  const bool early = FUSED && !fresh(1);
  if (early) {
    load_k(0, 0);
    load_k(1, 1);
    load_v(0, 0);
    load_v(1, 1);
  }
  if constexpr (FUSED) {
    fuse_wait(fc);
    __builtin_amdgcn_sched_barrier(0);
  }

  // stage the Q fragments: entry (t, ks, l) = pair t*16 + l%16, dims ks*32 + 8*(l/16) .. +7.
  // Their loads go out before the K/V loads (returns are in order per wavefront).
  // All of these loads are unconditional (entries past the group re-read a
  // valid one and are zeroed; a wave without tiles reads the chunk's first):
  // a branch around any of them would make the wait for Q below also wait for
  // every K/V load in flight.
  constexpr int QE = (NQ * KS * 64 + 64 * NWA - 1) / (64 * NWA);   // entries per thread
  const __amdgpu_buffer_rsrc_t qrs = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint16_t*>(p.q), 0,
                                                                        kMaxPassRows * p.ldq * 2, kRsrcWord3);
  u32x4 qv[QE];
#pragma unroll
  for (int j = 0; j < QE; ++j) {
    const int e = tid + j * 64 * NWA;
    const int ec = min(e, NQ * KS * 64 - 1);
    const int t = ec / (KS * 64), ks = (ec / 64) % KS, l = ec & 63;
    const int qh = qg * QP + t * 16 + (l & 15);
    const int qhc = min(qh, n_qh - 1);
    const int row = qhc / group, head = kvh * group + qhc % group;
    u32x4 v;
    if constexpr (FUSED)   // Q was written in this launch: device-scope load
      v = __builtin_amdgcn_raw_buffer_load_b128(qrs, ((d.row0 + row) * p.ldq + head * HD + ks * 32 + (l >> 4) * 8) * 2,
                                                0, kCachePolicyDevice);
    else
      v = *reinterpret_cast<const u32x4*>(p.q + (size_t)(d.row0 + row) * p.ldq + head * HD + ks * 32 + (l >> 4) * 8);
    qv[j] = (e < NQ * KS * 64 && qh < n_qh) ? v : u32x4{0u, 0u, 0u, 0u};
  }
  __builtin_amdgcn_sched_barrier(0);                // Q's loads, then both tiles' K, then V
  if (!early) {
    load_k(0, 0);
    load_k(1, 1);
    __builtin_amdgcn_sched_barrier(0);
    load_v(0, 0);
    load_v(1, 1);
  }
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

  // Not fused (the standalone kernel): the next pair's K is requested once
  // this pair's scores are computed and its V once this pair's V has been
  // multiplied, so a pair's loads are in flight during the previous pair's
  // work.  Fused (the decode launch) the loads stay at the top of each pair
  // (the early requests measured slower there).
  for (int it0 = 0; it0 < n_my; it0 += 2) {
    const int nt = min(2, n_my - it0);     // tiles in this pair (uniform)
    if (FUSED && it0 > 0) {
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
    if constexpr (!FUSED) {
      if (it0 + 2 < n_my) {                // uniform: the next pair's keys
        __builtin_amdgcn_sched_barrier(0);
        load_k(0, it0 + 2);
        load_k(1, it0 + 3);
        __builtin_amdgcn_sched_barrier(0);
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
    if constexpr (!FUSED) {
      if (it0 + 2 < n_my) {                // uniform: the next pair's values
        __builtin_amdgcn_sched_barrier(0);
        load_v(0, it0 + 2);
        load_v(1, it0 + 3);
        __builtin_amdgcn_sched_barrier(0);
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
  const __amdgpu_buffer_rsrc_t ors = __builtin_amdgcn_make_buffer_rsrc(
      p.out, 0, p.act_rows * p.n_heads * HD * 2, kRsrcWord3);
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
        const f32x4 a1 = a * linv_lds[q], b1 = b * linv_lds[q];
        if constexpr (FUSED) {   // read in this launch by the O-projection workers: device scope
          const u32x4 v = u32x4{pack_f16x2(a1[0], a1[1]), pack_f16x2(a1[2], a1[3]), pack_f16x2(b1[0], b1[1]),
                                pack_f16x2(b1[2], b1[3])};
          __builtin_amdgcn_raw_buffer_store_b128(v, ors, (int)act_index(d.row0 + row, head * HD + d0, p.act_rows) * 2, 0,
                                                 kCachePolicyDevice);
        } else {
          store_f16x8(p.out + act_index(d.row0 + row, head * HD + d0, p.act_rows), a1, b1);
        }
      }
    } else {
      *reinterpret_cast<f32x4*>(rec + q * HD + d0) = a;
      *reinterpret_cast<f32x4*>(rec + q * HD + d0 + 4) = b;
    }
  }
}

}  // namespace attn
}  // namespace pard
