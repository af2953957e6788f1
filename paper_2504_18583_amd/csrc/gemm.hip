// Skinny bf16 GEMM for decode-sized row counts, on gfx950 MFMA.
//
//   Y[r, n] = sum_k A[r, k] * W[n, k]            (W block-packed, A fp16)
//
// Decode streams every weight once per forward (Sec. 2.1: decoding is bound by
// reloading the weights), so the kernel is organised around the weight
// stream.  A workgroup owns S strips (16 output columns each) over the whole
// input dimension (the grid's last gate/up workgroup of 8-10 strips may own
// fewer, so that one round of workgroups covers the weight); its NW wavefronts
// split the input dimension, each one
// streaming its slice of the strips' 1 KiB blocks (one 16-byte load per lane,
// directly in the 16x16x32 MFMA B-operand layout) through a double-buffered
// register pipeline and accumulating MT 16x16 fp32 tiles.  Activation rows
// (<= 16*MT) are the A operand, in fp16; the weights (bf16 values kept in fp16
// encoding) feed v_mfma_f32_16x16x32_f16 directly.
//
// The wavefront partials are summed in LDS in wave order, so results are
// deterministic; the split depends only on the weight shape, so a row's result
// does not depend on how many other rows are in the pass.  No workgroup ever
// waits for another one.
//
// Shapes with few strips also split the input dimension over the grid's y
// dimension (P contiguous ranges of k-blocks), so that narrow GEMMs still
// occupy every CU and one activation fragment feeds several strips.  Each
// workgroup stores its fp32 partial tile and counts itself in on the tile's
// counter; the last of the P to arrive adds the P partials in range order
// (the same order whichever workgroup is last) and runs the epilogue, then
// resets the counter for the next launch.
//
// Epilogues fuse the surrounding element-wise work of a Llama block:
//   EPI_QKV     RMSNorm row scale (A holds x*g in fp16, written by the
//               producer; 1/rms comes from the producer's per-tile sums of
//               squares), bias, rotate-half RoPE on Q/K, Q to an fp16 buffer,
//               K (16-key MFMA fragments) and V (32-key blocks, transposed)
//               to the fp16 cache.
//   EPI_RESID   x += Y (O-projection, down-projection), plus fp16(x * g_next)
//               and per-tile row sums of squares for the next normalised GEMM.
//   EPI_SWIGLU  RMSNorm row scale, h = silu(gate) * up, fp16 (each strip
//               holds 8 gate and the 8 matching up columns).
//   EPI_LOGITS  final RMSNorm scale, fp32 logits and per-tile (max, argmax).
// k_lm_tail then reduces the tiles per row (lowest id on ties) and runs the
// step tail: candidates for a draft pass; greedy prefix acceptance, KV
// rollback and next-pass staging for a verify pass.
#include "attn_tile.h"
#include "pard_internal.h"

#include <hip/hip_ext.h>

#include <algorithm>
#include <climits>
#include <map>
#include <type_traits>

namespace pard {
namespace {

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));



constexpr int kRsrcWord3 = 0x00020000;   // buffer descriptor word 3 for gfx9-family raw buffers
constexpr int kCachePolicyNT = 2;        // non-temporal: weights are streamed once
constexpr int kWaitVmcnt0 = 0x0F70;      // s_waitcnt vmcnt(0), expcnt and lgkmcnt not waited for

// Sum over the 16 lanes of a DPP row (lanes 16g .. 16g+15), fixed order:
// quad_perm swaps (1 0 3 2), (2 3 0 1), then half-row and row mirrors.
__device__ __forceinline__ float sum16(float x) {
  x += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), 0xB1, 0xF, 0xF, false));
  x += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), 0x4E, 0xF, 0xF, false));
  x += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), 0x141, 0xF, 0xF, false));
  x += __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), 0x140, 0xF, 0xF, false));
  return x;
}

__device__ __forceinline__ bool better(float v, int i, float bv, int bi) {
  return v > bv || (v == bv && i < bi);
}

// Wavefront reductions and scan in a fixed order (results do not depend on timing).
__device__ __forceinline__ float wave_sum(float v) {
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off);
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
  for (int off = 32; off > 0; off >>= 1) v = fmaxf(v, __shfl_xor(v, off));
  return v;
}
__device__ __forceinline__ float wave_incl_scan(float v, int lane) {
  for (int off = 1; off < 64; off <<= 1) {
    const float o = __shfl_up(v, off);
    if (lane >= off) v += o;
  }
  return v;
}

// Input iterations per wavefront that a fused gate/up tile may take from LDS.
constexpr int kGuPreMax = 8;

// One workgroup tile of the skinny GEMM: strips [tile*S, tile*S + S) over the
// input range `split` of n_split, computed by the first nw wavefronts of the
// workgroup; red is the [nw][S*MT*256] float LDS of the wave reduction.  With
// FUSED (the QKV GEMM of a launch that also carries the attention reading its
// output) the Q / K / V stores are device-scope, so that workgroups on other
// XCDs of the same launch read them after the count-in.  With PM = 1 (the gate/up
// tile of such a launch: one row tile, one input range, four wavefronts) the
// first `pre` iterations of each wavefront take their weights from LDS, the
// first pre_d of them from pre_lds and the rest from pre_stat (gu_preload put
// them there; the caller has waited for its loads), the
// first global weight stages are requested before the tile waits for the O
// workers (fc), and the activations and row sums they wrote in this launch
// are read at device scope (one acquire fence per workgroup measured 8B/1B
// 3.511 ms against 3.456, one per wavefront 3.757), and h is stored at device
// scope.  With PM = 2 (the down projection of such a launch, one strip per
// tile) the first weight stages are requested before the tile waits for every
// gate/up tile (fc), and h and the residual x, written in this launch, are
// read at device scope.  The arithmetic and its order are those of the
// unfused tile.
template <int MT, int S, int EPI, bool FUSED = false, int PM = 0>
__device__ __forceinline__ void gemm_tile(const GemmArgs& p, const int tile, const unsigned split, const int n_split,
                                          const int nw, float* red, const FuseCtl* fc = nullptr,
                                          const uint32_t* pre_lds = nullptr, const int pre = 0,
                                          const uint32_t* pre_stat = nullptr, const int pre_d = 0,
                                          const int red_stride = 0) {
  static_assert(PM != 1 || (MT == 1 && EPI == EPI_SWIGLU && S < 8), "preloaded tiles: one row tile of gate/up, not ragged");
  static_assert(PM != 2 || (MT == 1 && EPI == EPI_RESID && S == 1), "fused down tiles: one row tile, one strip");
  constexpr int NE = S * MT * 256;   // elements of one workgroup tile
  constexpr int NJ = S * MT;         // elements per thread in the epilogue (first 256 threads)
  // k-blocks per pipeline stage: 8 KiB of W per wave (smaller for prefill-sized row counts)
  constexpr int U = MT >= 3 ? 2 : ((8 / S) > 0 ? 8 / S : 1);
  __shared__ float rs_s[MT * 16];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // uniform per wavefront

  // input range of this workgroup: k-blocks [kb0, kb0 + kb_n)
  const int kb0 = split * p.kb_split;
  const int kb_n = min(p.kb_split, p.kb_total - kb0);
  // wave w streams k-blocks kb0 + w, kb0 + w + nw, ...: at any time the
  // workgroup reads nw consecutive k-blocks of each strip
  const int n_it = (kb_n - wave + nw - 1) / nw;

  f32x4 acc[S][MT];
#pragma unroll
  for (int s = 0; s < S; ++s)
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) acc[s][mt] = f32x4{0.f, 0.f, 0.f, 0.f};

  // Raw buffer loads: a per-matrix descriptor, a constant per-lane VGPR offset
  // and a scalar per-iteration offset, so the prefetch needs no VGPR address
  // arithmetic (which would otherwise force waits on in-flight loads), and
  // every access is bounds-checked by the hardware.
  // W is k-block-major: block (kb, strip) sits at (kb * n_strips + strip) KiB.
  // A gate/up workgroup of 8 or more strips may be the grid's last, with
  // fewer strips than S (ragged): its missing strips re-read its last strip
  // (cache hits) and store nothing.
  constexpr bool RAGGED = EPI == EPI_SWIGLU && MT == 1 && S >= 8;
  const int n_strips = p.n_strips;
  const int s_last = RAGGED ? min(S - 1, n_strips - 1 - tile * S) : S - 1;
  const __amdgpu_buffer_rsrc_t wrs = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(p.W), 0, (int)min((size_t)n_strips * p.kb_total * 1024, (size_t)0x7fffffff), kRsrcWord3);
  const int w_voff = (tile * S * 64 + lane) * 16;

  // Two register stages of U k-blocks each: loads of stage i+1 are in flight
  // while stage i feeds the MFMAs.  Iterations past the wave's range are
  // clamped (cache hits) and their A fragment is zeroed.
  u32x4 w0[U][S], a0[U][MT], w1[U][S], a1[U][MT];
  auto load_w = [&](u32x4 (&w)[U][S], int its) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int kb = kb0 + wave + min(its + u, n_it - 1) * nw;
#pragma unroll
      for (int s = 0; s < S; ++s)
        w[u][s] = __builtin_amdgcn_raw_buffer_load_b128(wrs, w_voff, (kb * n_strips + (RAGGED ? min(s, s_last) : s)) * 1024,
                                                        kCachePolicyNT);
    }
  };

  constexpr bool LM = EPI == EPI_LOGITS;              // rows are the pass's lm rows
  constexpr bool NORM = EPI != EPI_RESID;             // A is RMS-normalised: rows need 1/rms

  // 1/rms per row from the producer's per-tile sums of squares: 16 threads per
  // row, fixed summation order.  For one row tile the loads of the first 256
  // tiles are issued ahead of the weight stream (ss_issue) and summed just
  // before the first MFMAs (ss_finish): loads complete in issue order, so
  // waiting for them would otherwise also wait for every weight load in
  // flight and empty the pipeline.
  float ss_part[16];
  auto ss_issue = [&](int row) {
#pragma unroll
    for (int u = 0; u < 16; ++u) {
      // unconditional loads (a tile index past the end re-reads the last
      // tile and is dropped when summed), so none waits behind a branch
      const int q = (tid & 15) + 16 * u;
      if constexpr (PM)   // written by the O workers of this launch: device scope
        ss_part[u] = __hip_atomic_load(p.ss_in + (size_t)row * p.ss_stride + min(q, p.ss_tiles - 1), __ATOMIC_RELAXED,
                                       __HIP_MEMORY_SCOPE_AGENT);
      else
        ss_part[u] = p.ss_in[(size_t)row * p.ss_stride + min(q, p.ss_tiles - 1)];
    }
  };
  auto ss_finish = [&](int row) {
    float t = 0.f;
#pragma unroll
    for (int u = 0; u < 16; ++u) t += (tid & 15) + 16 * u < p.ss_tiles ? ss_part[u] : 0.f;
    for (int q0 = (tid & 15) + 256; q0 < p.ss_tiles; q0 += 256) {
      float part[16];
#pragma unroll
      for (int u = 0; u < 16; ++u) {
        const int q = q0 + 16 * u;
        if constexpr (PM)
          part[u] = q < p.ss_tiles ? __hip_atomic_load(p.ss_in + (size_t)row * p.ss_stride + q, __ATOMIC_RELAXED,
                                                       __HIP_MEMORY_SCOPE_AGENT) : 0.f;
        else
          part[u] = q < p.ss_tiles ? p.ss_in[(size_t)row * p.ss_stride + q] : 0.f;
      }
#pragma unroll
      for (int u = 0; u < 16; ++u) t += part[u];
    }
    t += __shfl_xor(t, 8);
    t += __shfl_xor(t, 4);
    t += __shfl_xor(t, 2);
    t += __shfl_xor(t, 1);
    if ((tid & 15) == 0) rs_s[tid >> 4] = 1.0f / sqrtf(t * p.inv_k + p.eps);
  };
  // thread tid (< 256) of the epilogue owns, for j = s*MT + mt, element
  // (row, col) below; its epilogue operands are fetched while the weights stream
  const bool epi = tid < 256;
  const int ew = tid >> 6;
  const int rsub = (lane >> 4) * 4 + ew;
  const int csub = lane & 15;

  // Per-lane reads of the pass descriptor are issued first, for the same
  // reason: lm source rows (A fragment rows, row-scale rows) and, for QKV, the
  // position and sequence slot of each epilogue row.  Entries past the pass
  // are read (in bounds) but never used.
  const FwdDesc* dp = p.desc;
  int lm_a[MT], e_pos[MT], e_slot[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    lm_a[mt] = LM ? dp->lm_src[mt * 16 + (lane & 15)] : 0;
    e_pos[mt] = EPI == EPI_QKV ? dp->pos[mt * 16 + rsub] : 0;
    e_slot[mt] = EPI == EPI_QKV ? dp->slot[mt * 16 + rsub] : 0;
  }
  const int lm_ss = LM ? dp->lm_src[(tid & 255) >> 4] : 0;
  // rows of a pass's activations need no descriptor (rows past the pass read
  // unused sums and are never stored)
  if constexpr (NORM && !LM && MT == 1 && !PM) {
    if (tid < 256) ss_issue(tid >> 4);
  }
  __builtin_amdgcn_sched_barrier(0);

  // The weight stream does not depend on the pass: its first stage is in
  // flight before the pass descriptor's scalar fields are read.  It is loaded
  // unconditionally (a wave with no k-block of its own, n_it = 0, reads the
  // range's last one and never uses it): a branch around it would make every
  // later wait on an earlier load wait for the whole stage too.
  const int its0 = PM == 1 ? pre : 0;   // the first iteration streamed from memory
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int kb = kb0 + min(wave + min(its0 + u, max(n_it - 1, 0)) * nw, kb_n - 1);
#pragma unroll
    for (int s = 0; s < S; ++s)
      w0[u][s] = __builtin_amdgcn_raw_buffer_load_b128(wrs, w_voff, (kb * n_strips + (RAGGED ? min(s, s_last) : s)) * 1024,
                                                       kCachePolicyNT);
  }
  __builtin_amdgcn_sched_barrier(0);

  const int row_count = LM ? dp->n_lm : dp->n_rows;
  const int ss_row = LM ? ((tid & 255) >> 4 < row_count ? lm_ss : 0) : (tid & 255) >> 4;
  if constexpr (LM && MT == 1) {
    if (tid < 256) ss_issue(ss_row);              // lm rows read their source row's sums
  }

  // A fragment of this lane: row (lane % 16) of each M tile, 8 columns at
  // 8*(lane/16); A is k-blocked, so k-block kb of all rows is one contiguous
  // run at kb * act_rows * 64 bytes.  Rows past the pass get an offset
  // beyond the buffer: the hardware returns zeros for them without a memory
  // access.  lm rows read their source row.
  const __amdgpu_buffer_rsrc_t ars = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(p.A), 0, p.act_rows * p.lda * 2, kRsrcWord3);
  constexpr int kOutOfRange = 0x7FFFFFF0;
  int a_voff[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    const int r = mt * 16 + (lane & 15);
    const int src = r < row_count ? (LM ? lm_a[mt] : r) : 0;
    a_voff[mt] = r < row_count ? src * 64 + (lane >> 4) * 16 : kOutOfRange;
  }
  auto load_a = [&](u32x4 (&a)[U][MT], int its) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int kb = kb0 + wave + min(its + u, n_it - 1) * nw;
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
        a[u][mt] = __builtin_amdgcn_raw_buffer_load_b128(ars, a_voff[mt], kb * (p.act_rows * 64),
                                                         PM ? attn::kCachePolicyDevice : 0);
    }
  };
  auto load = [&](u32x4 (&w)[U][S], u32x4 (&a)[U][MT], int its) {
    load_w(w, its);
    load_a(a, its);
  };

  float e0[NJ], e1[NJ];
  float2 e2[NJ];
  auto prefetch_epilogue = [&]() {
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const int s = j / MT, mt = j % MT;
      const int row = mt * 16 + rsub;
      const int n = (tile * S + s) * 16 + csub;
      e0[j] = 0.f;
      e1[j] = 0.f;
      e2[j] = float2{1.f, 0.f};
      if constexpr (EPI == EPI_RESID) {
        if (epi && row < row_count) {
          if constexpr (PM == 2)   // written by the O workers of this launch
            e0[j] = __hip_atomic_load(p.x + (size_t)row * p.ldx + n, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
          else
            e0[j] = p.x[(size_t)row * p.ldx + n];
          e1[j] = p.g_next[n];
        }
      } else if constexpr (EPI == EPI_QKV) {
        if (epi && p.bias) e0[j] = p.bias[n];
        if (epi && row < row_count && n < p.q_dim + p.kv_dim)
          e2[j] = p.rope[(size_t)e_pos[mt] * (p.hd / 2) + ((n % p.hd) >> 1)];
      }
    }
  };
  auto compute = [&](const u32x4 (&w)[U][S], const u32x4 (&a)[U][MT], int its) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const bool live = its + u < n_it;
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        const u32x4 av = live ? a[u][mt] : u32x4{0u, 0u, 0u, 0u};
#pragma unroll
        for (int s = 0; s < S; ++s)
          acc[s][mt] = __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, av),
                                                              __builtin_bit_cast(f16x8, w[u][s]), acc[s][mt], 0, 0, 0);
      }
    }
  };

  // several row tiles: the same sums, loaded and summed in one go
  auto row_scales = [&]() {
    if (tid < 256) {
      for (int r = tid >> 4; r < MT * 16; r += 16) {
        const int row = r < row_count ? (LM ? dp->lm_src[r] : r) : 0;
        float t = 0.f;
        for (int q0 = tid & 15; q0 < p.ss_tiles; q0 += 256) {
          float part[16];
#pragma unroll
          for (int u = 0; u < 16; ++u) {
            const int q = q0 + 16 * u;
            part[u] = q < p.ss_tiles ? p.ss_in[(size_t)row * p.ss_stride + q] : 0.f;
          }
#pragma unroll
          for (int u = 0; u < 16; ++u) t += part[u];
        }
        t += __shfl_xor(t, 8);
        t += __shfl_xor(t, 4);
        t += __shfl_xor(t, 2);
        t += __shfl_xor(t, 1);
        if ((tid & 15) == 0) rs_s[r] = 1.0f / sqrtf(t * p.inv_k + p.eps);
      }
    }
  };

  // sched_barrier keeps the compiler from sinking the prefetch next to its use
  if constexpr (PM == 2) {
    int its = 0;
    load_w(w1, its + U);                                // the second stage, before the wait
    __builtin_amdgcn_sched_barrier(0);
    attn::fuse_wait_on<kFuseLanes>(fc->counters + 3 * kFuseLanes * kFuseStride, fc->gu_tiles, fc->err);
    load_a(a0, its);
    load_a(a1, its + U);
    __builtin_amdgcn_sched_barrier(0);
    prefetch_epilogue();
    __builtin_amdgcn_sched_barrier(0);
    while (its + 2 * U < n_it) {
      compute(w0, a0, its);
      __builtin_amdgcn_sched_barrier(0);
      load(w0, a0, its + 2 * U);
      __builtin_amdgcn_sched_barrier(0);
      compute(w1, a1, its + U);
      __builtin_amdgcn_sched_barrier(0);
      load(w1, a1, its + 3 * U);
      __builtin_amdgcn_sched_barrier(0);
      its += 2 * U;
    }
    compute(w0, a0, its);
    if (its + U < n_it) compute(w1, a1, its + U);     // uniform
  } else if constexpr (PM == 1) {
    int its = pre;
    load_w(w1, its + U);                                // the second stage, before the wait
    __builtin_amdgcn_sched_barrier(0);
    attn::fuse_wait_on<kFuseLanes>(fc->counters + 2 * kFuseLanes * kFuseStride, fc->n_odone, fc->err);
    if (tid < 256) ss_issue(tid >> 4);
    load_a(a0, its);
    load_a(a1, its + U);
    // A of the preloaded iterations (iterations past `pre` re-read the last
    // one and are never used)
    u32x4 ap[kGuPreMax];
#pragma unroll
    for (int i = 0; i < kGuPreMax; ++i)
      ap[i] = __builtin_amdgcn_raw_buffer_load_b128(ars, a_voff[0], (kb0 + wave + min(i, max(pre - 1, 0)) * nw) *
                                                    (p.act_rows * 64), attn::kCachePolicyDevice);
    __builtin_amdgcn_sched_barrier(0);
    if (tid < 256) ss_finish(ss_row);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int i = 0; i < kGuPreMax; ++i) {
      if (i < pre) {                                    // uniform
#pragma unroll
        for (int s = 0; s < S; ++s) {
          const uint32_t* wb = i < pre_d ? pre_lds + ((wave * pre_d + i) * S + s) * 256
                                         : pre_stat + ((wave * (pre - pre_d) + i - pre_d) * S + s) * 256;
          const u32x4 wl = *reinterpret_cast<const u32x4*>(wb + lane * 4);
          acc[s][0] = __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, ap[i]),
                                                             __builtin_bit_cast(f16x8, wl), acc[s][0], 0, 0, 0);
        }
      }
    }
    __builtin_amdgcn_sched_barrier(0);
    while (its + 2 * U < n_it) {
      compute(w0, a0, its);
      __builtin_amdgcn_sched_barrier(0);
      load(w0, a0, its + 2 * U);
      __builtin_amdgcn_sched_barrier(0);
      compute(w1, a1, its + U);
      __builtin_amdgcn_sched_barrier(0);
      load(w1, a1, its + 3 * U);
      __builtin_amdgcn_sched_barrier(0);
      its += 2 * U;
    }
    compute(w0, a0, its);
    if (its + U < n_it) compute(w1, a1, its + U);     // uniform
  } else if (n_it > 0) {
    int its = 0;
    load_a(a0, its);
    __builtin_amdgcn_sched_barrier(0);
    if constexpr (NORM && MT > 1) row_scales();     // overlaps the first weight loads
    load(w1, a1, its + U);
    __builtin_amdgcn_sched_barrier(0);
    prefetch_epilogue();
    __builtin_amdgcn_sched_barrier(0);
    if constexpr (NORM && MT == 1) {
      if (tid < 256) ss_finish(ss_row);
    }
    __builtin_amdgcn_sched_barrier(0);
    // One exit per pair of stages, at the loop's top: with an exit between
    // the two halves the compiler's wait at the top covered every load in
    // flight (draining the pipeline once per pair); with one exit it waits
    // only for the stage it computes.  The last two stages are computed after
    // the loop (loads past the range are clamped: at most one stage of them).
    while (its + 2 * U < n_it) {
      compute(w0, a0, its);
      __builtin_amdgcn_sched_barrier(0);
      load(w0, a0, its + 2 * U);
      __builtin_amdgcn_sched_barrier(0);
      compute(w1, a1, its + U);
      __builtin_amdgcn_sched_barrier(0);
      load(w1, a1, its + 3 * U);
      __builtin_amdgcn_sched_barrier(0);
      its += 2 * U;
    }
    compute(w0, a0, its);
    if (its + U < n_it) compute(w1, a1, its + U);     // uniform
  } else {
    if constexpr (NORM && MT > 1) row_scales();
    if constexpr (NORM && MT == 1) {
      if (tid < 256) ss_finish(ss_row);
    }
    prefetch_epilogue();
  }

  // ---- workgroup reduction over the NW input-dimension slices (wave order) ----
  const int rs = red_stride > 0 ? red_stride : NE;    // floats between the wavefronts' partial tiles
#pragma unroll
  for (int s = 0; s < S; ++s)
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int i = 0; i < 4; ++i) red[wave * rs + ((s * MT + mt) * 4 + i) * 64 + lane] = acc[s][mt][i];

  __syncthreads();

  // the first four wavefronts run the epilogue; all waves stay until the end
  // so that every barrier below is reached by the whole workgroup
  float v[NJ];
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    const int e = j * 256 + (tid & 255);
    float t = red[e];
    for (int w = 1; w < nw; ++w) t += red[w * rs + e];
    v[j] = t;
  }

  // ---- split input dimension: the last workgroup of the tile to finish sums the partials ----
  // Partials are stored and loaded at device scope (written through to, and
  // read from, the level shared by all XCDs), so the count needs no cache
  // write-back or invalidation: each wavefront waits until its stores are
  // complete before the workgroup counts itself in.
  if (n_split > 1) {
    __shared__ int last_s;
    float* part = p.part + (size_t)tile * n_split * NE;
    if (epi) {
#pragma unroll
      for (int j = 0; j < NJ; ++j)
        __hip_atomic_store(part + (size_t)split * NE + j * 256 + tid, v[j], __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
    }
    __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
    __syncthreads();
    if (tid == 0) {
      const int prev = __hip_atomic_fetch_add(p.counters + tile, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      last_s = prev == n_split - 1;
      if (prev == n_split - 1) __hip_atomic_store(p.counters + tile, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    __syncthreads();
    if (!last_s) return;    // uniform over the workgroup
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const int e = j * 256 + (tid & 255);
      float t = 0.f;
      for (int q = 0; q < n_split; ++q)
        t += __hip_atomic_load(part + (size_t)q * NE + e, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      v[j] = t;
    }
  }

  [[maybe_unused]] bool bad = false;
  if constexpr (EPI == EPI_QKV) {
    if (!epi) return;   // no barrier follows in this epilogue
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const int s = j / MT, mt = j % MT;
      const int row = mt * 16 + rsub;
      const int n = (tile * S + s) * 16 + csub;
      float y = v[j] * rs_s[row] + e0[j];            // + bias
      // rotary partner column (n ^ 1) is in lane l ^ 1 (DPP quad swap)
      const float partner = __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, y), 0xB1, 0xF,
                                                                               0xF, false));
      if (row < row_count) {
        const int pos = e_pos[mt];
        const size_t cache = (size_t)e_slot[mt] * p.kv_seq_stride;
        if (n < p.q_dim + p.kv_dim) {
          const float2 cs = e2[j];                     // rotary (cos, sin) of (pos, pair)
          y = (n & 1) ? (y * cs.x + partner * cs.y) : (y * cs.x - partner * cs.y);
        }
        const uint16_t b = f16_flagged(y, bad);
        uint16_t* dst;
        if (n < p.q_dim) {
          dst = p.out + (size_t)row * p.ld_out + n;
        } else if (n < p.q_dim + p.kv_dim) {
          const int c = n - p.q_dim;
          dst = p.kc + cache + (size_t)(c / p.hd) * p.cap * p.hd + k_index(pos, c % p.hd, p.hd);
        } else {
          const int c = n - p.q_dim - p.kv_dim;
          const size_t blk = (size_t)(c / p.hd) * (p.cap / 32) + (pos >> 5);
          dst = p.vc + cache + (blk * p.hd + (c % p.hd)) * 32 + v_slot(pos & 31);
        }
        if constexpr (FUSED)
          __hip_atomic_store(dst, b, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        else
          *dst = b;
      }
    }
    flag_range(bad, p.ovf);
  } else if constexpr (EPI == EPI_RESID) {
    if (!epi) return;   // no barrier follows in this epilogue
    float sq[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) sq[mt] = 0.f;
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const int s = j / MT, mt = j % MT;
      const int row = mt * 16 + rsub;
      const int n = (tile * S + s) * 16 + csub;
      if (row < row_count) {
        const size_t o = (size_t)row * p.ldx + n;
        const float xn = e0[j] + v[j];                 // residual + projection
        p.x[o] = xn;
        p.xg[act_index(row, n, p.act_rows)] = f16_flagged(xn * e1[j], bad);
        sq[mt] += xn * xn;
      }
    }
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      const float t = sum16(sq[mt]);
      if (csub == 0) p.ss_out[(size_t)(mt * 16 + rsub) * p.ss_stride + tile] = t;
    }
    flag_range(bad, p.ovf);
  } else if constexpr (EPI == EPI_SWIGLU) {
    // a strip holds 8 gate columns then the 8 up columns of the same features:
    // the up value of column csub < 8 is in lane ^ 8 (same row)
    if (!epi) return;   // whole wavefronts; no barrier follows in this epilogue
#pragma unroll
    for (int s = 0; s < S; ++s)
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        const int row = mt * 16 + rsub;
        const float gt = v[s * MT + mt] * rs_s[row];
        // lane l ^ 8 of the row of 16 (DPP row rotate by 8)
        const float up = __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, gt), 0x128, 0xF,
                                                                            0xF, false));
        const float h = gt / (1.0f + expf(-gt)) * up;
        const int f = (tile * S + s) * 8 + csub;
        if (csub < 8 && row < row_count && s <= s_last) {
          if constexpr (PM == 1)   // read by the down tiles of this launch: device scope
            __hip_atomic_store(p.out + act_index(row, f, p.act_rows), f16_flagged(h, bad), __ATOMIC_RELAXED,
                               __HIP_MEMORY_SCOPE_AGENT);
          else
            p.out[act_index(row, f, p.act_rows)] = f16_flagged(h, bad);
        }
      }
    flag_range(bad, p.ovf);
  } else {  // EPI_LOGITS
    constexpr int TW = S * 16;
    __syncthreads();   // everyone is done reading red; it becomes the [row][col] tile
    if (epi) {
#pragma unroll
      for (int j = 0; j < NJ; ++j) {
        const int s = j / MT, mt = j % MT;
        const int row = mt * 16 + rsub;
        const int c = s * 16 + csub;
        const float val = v[j] * rs_s[row];
        red[row * TW + c] = val;
        if (row < row_count) p.logits[(size_t)row * p.vocab + tile * TW + c] = val;
      }
    }
    __syncthreads();
    if (!epi) return;
    for (int r = ew; r < row_count; r += 4) {
      float bv = -INFINITY;
      int bi = INT_MAX;
      for (int c = lane; c < TW; c += 64) {
        const float x = red[r * TW + c];
        if (better(x, c, bv, bi)) { bv = x; bi = c; }
      }
      for (int off = 32; off > 0; off >>= 1) {
        const float ov = __shfl_xor(bv, off);
        const int oi = __shfl_xor(bi, off);
        if (better(ov, oi, bv, bi)) { bv = ov; bi = oi; }
      }
      if (lane == 0) {
        p.amax_val[(size_t)r * p.amax_stride + tile] = bv;
        p.amax_idx[(size_t)r * p.amax_stride + tile] = (bi == INT_MAX) ? INT_MAX : tile * TW + bi;
      }
      if (p.samp_k > 0.f) {         // sampling: the tile's softmax weight relative to its max
        float sw = 0.f;
        for (int c = lane; c < TW; c += 64) sw += __builtin_amdgcn_exp2f((red[r * TW + c] - bv) * p.samp_k);
        sw = wave_sum(sw);
        if (lane == 0) p.amax_sum[(size_t)r * p.amax_stride + tile] = sw;
      }
    }
  }
}

template <int MT, int S, int EPI>
__global__ __launch_bounds__(512) void k_gemm(const GemmArgs p) {
  extern __shared__ float red[];     // [NW][NE]
  gemm_tile<MT, S, EPI>(p, blockIdx.x, blockIdx.y, gridDim.y, blockDim.x >> 6, red);
}

// O-projection units of a fused decode-layer launch (one row tile, EPI_RESID,
// one strip per unit, the whole input range): NU units of this worker
// starting at strip u0.  Wavefront v of the eight holds k-blocks v, v + 8, ...
// (KI of them; past the input range it re-reads the last one and never uses
// it).  Every weight block is requested before the wait for the attention
// workgroups, so the weights stream while the attention runs; the attention
// output (written in this launch) is then read at device scope.  The eight
// wavefront partials are summed in wave order, then the residual epilogue of
// gemm_tile: x += Y, fp16(x * g_next) and the strip's row sums of squares.
template <int KI, int NU, bool GUF, class Pre>
__device__ __forceinline__ void o_units(const GemmArgs& p, const FuseCtl& f, const int u0, float* red, Pre&& preload) {
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int n_strips = p.n_strips, kb_total = p.kb_total;
  const __amdgpu_buffer_rsrc_t wrs = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(p.W), 0, (int)min((size_t)n_strips * kb_total * 1024, (size_t)0x7fffffff), kRsrcWord3);
  u32x4 wv[NU][KI];
#pragma unroll
  for (int i = 0; i < KI; ++i) {
    const int kb = min(wave + 8 * i, kb_total - 1);
#pragma unroll
    for (int j = 0; j < NU; ++j)
      wv[j][i] = __builtin_amdgcn_raw_buffer_load_b128(wrs, ((u0 + j) * 64 + lane) * 16, kb * n_strips * 1024,
                                                       kCachePolicyNT);
  }
  __builtin_amdgcn_sched_barrier(0);
  preload();                                         // gate/up weights into LDS, behind the O weights
  __builtin_amdgcn_sched_barrier(0);
  // epilogue element of this thread: unit ej, row rsub, column csub of the
  // strip (the MFMA output layout; threads < 256 * NU)
  const int row_count = p.desc->n_rows;
  const bool epi = tid < 256 * NU;
  const int ej = min(tid >> 8, NU - 1);
  const int rsub = (lane >> 4) * 4 + ((tid & 255) >> 6), csub = lane & 15;
  const int n = (u0 + ej) * 16 + csub;
  float x_old = 0.f, g = 0.f;
  if (epi && rsub < row_count) {
    x_old = p.x[(size_t)rsub * p.ldx + n];
    g = p.g_next[n];
  }
  __builtin_amdgcn_sched_barrier(0);
  attn::fuse_wait_on<1>(f.counters + (kFuseLanes + blockIdx.x % kFuseLanes) * kFuseStride, f.n_cons, f.err);
  __builtin_amdgcn_sched_barrier(0);
  // A fragment of this lane: row lane % 16, 8 columns at 8 * (lane / 16) of
  // each k-block; rows past the pass read zeros without a memory access
  constexpr int kOutOfRange = 0x7FFFFFF0;
  const __amdgpu_buffer_rsrc_t ars = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(p.A), 0, p.act_rows * p.lda * 2, kRsrcWord3);
  const int a_voff = (lane & 15) < row_count ? (lane & 15) * 64 + (lane >> 4) * 16 : kOutOfRange;
  u32x4 av[KI];
#pragma unroll
  for (int i = 0; i < KI; ++i)
    av[i] = __builtin_amdgcn_raw_buffer_load_b128(ars, a_voff, min(wave + 8 * i, kb_total - 1) * (p.act_rows * 64),
                                                  attn::kCachePolicyDevice);
  f32x4 acc[NU];
#pragma unroll
  for (int j = 0; j < NU; ++j) acc[j] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int i = 0; i < KI; ++i) {
    const u32x4 a = wave + 8 * i < kb_total ? av[i] : u32x4{0u, 0u, 0u, 0u};
#pragma unroll
    for (int j = 0; j < NU; ++j)
      acc[j] = __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, a), __builtin_bit_cast(f16x8, wv[j][i]),
                                                      acc[j], 0, 0, 0);
  }
#pragma unroll
  for (int j = 0; j < NU; ++j)
#pragma unroll
    for (int i = 0; i < 4; ++i) red[(wave * NU + j) * 256 + i * 64 + lane] = acc[j][i];
  __syncthreads();
  if (!epi) return;   // whole wavefronts; no barrier follows
  float v = red[ej * 256 + (tid & 255)];
  for (int w = 1; w < 8; ++w) v += red[(w * NU + ej) * 256 + (tid & 255)];
  float sq = 0.f;
  bool bad = false;
  if (rsub < row_count) {
    const float xn = x_old + v;                      // residual + projection
    if constexpr (GUF)   // read by the down tiles of this launch: device scope
      __hip_atomic_store(p.x + (size_t)rsub * p.ldx + n, xn, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    else
      p.x[(size_t)rsub * p.ldx + n] = xn;
    const uint16_t h = f16_flagged(xn * g, bad);
    if constexpr (GUF)   // read by the gate/up tiles of this launch: device scope
      __hip_atomic_store(p.xg + act_index(rsub, n, p.act_rows), h, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    else
      p.xg[act_index(rsub, n, p.act_rows)] = h;
    sq = xn * xn;
  }
  const float t = sum16(sq);
  if (csub == 0) {
    if constexpr (GUF)
      __hip_atomic_store(p.ss_out + (size_t)rsub * p.ss_stride + u0 + ej, t, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    else
      p.ss_out[(size_t)rsub * p.ss_stride + u0 + ej] = t;
  }
  flag_range(bad, p.ovf);
}

// The O units of worker w (see FuseCtl), if it has any; `preload` runs once
// in any case (after the O weight requests when there are units).  With GUF
// (gate/up in the launch) a worker with units counts itself in once its
// stores are complete.
template <int KI, bool GUF, class Pre>
__device__ __forceinline__ void o_part(const GemmArgs& p, const FuseCtl& f, const int w, float* red, Pre&& preload) {
  if (w < f.o_two) {
    o_units<KI, 2, GUF>(p, f, 2 * w, red, preload);
  } else if (f.o_two + w < f.o_units) {
    o_units<KI, 1, GUF>(p, f, f.o_two + w, red, preload);
  } else {
    preload();
    return;
  }
  if constexpr (GUF) {
    __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);          // this wavefront's stores are complete
    __syncthreads();
    if (threadIdx.x == 0)
      __hip_atomic_fetch_add(f.counters + (2 * kFuseLanes + blockIdx.x % kFuseLanes) * kFuseStride, 1,
                             __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

// Gate/up weights of tile `tile` for input iterations [i0, i1) of
// wavefronts 0-3 (k-blocks w + 4i, as gemm_tile streams them), loaded
// straight into LDS (1 KiB blocks, lane-ordered) with no registers held:
// iterations below pre_d at dyn [w][i][strip], the others (STAT) at stat
// [w][i - pre_d][strip] for a workgroup of `pre` iterations; called by
// wavefronts 0-3, each for its own blocks.  Every load's LDS target derives
// from one LDS object, so the compiler's LDS-DMA waits stay precise.
template <int S, bool STAT>
__device__ __forceinline__ void gu_preload(const GemmArgs& p, const int tile, const int i0, const int i1,
                                           const int pre, const int pre_d, uint32_t* dyn, uint32_t* stat) {
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const __amdgpu_buffer_rsrc_t wrs = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(p.W), 0, (int)min((size_t)p.n_strips * p.kb_total * 1024, (size_t)0x7fffffff), kRsrcWord3);
  const int voff = (tile * S * 64 + lane) * 16;
  for (int i = i0; i < min(i1, pre_d); ++i) {
    const int kb = wave + 4 * i;                     // < kb_total: pre <= kb_total / 4 (host)
#pragma unroll
    for (int s = 0; s < S; ++s)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          wrs, (__attribute__((address_space(3))) void*)(dyn + ((wave * pre_d + i) * S + s) * 256), 16, voff,
          (kb * p.n_strips + s) * 1024, 0, kCachePolicyNT);
  }
  if constexpr (STAT) {
    for (int i = max(i0, pre_d); i < i1; ++i) {
      const int kb = wave + 4 * i;
#pragma unroll
      for (int s = 0; s < S; ++s)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(
            wrs, (__attribute__((address_space(3))) void*)(stat + ((wave * (pre - pre_d) + i - pre_d) * S + s) * 256),
            16, voff, (kb * p.n_strips + s) * 1024, 0, kCachePolicyNT);
    }
  }
}

// Static LDS of the one-launch layer: the attention arrays of its attention
// workgroups, and in the others (and in those after their attention) the last
// preloaded gate/up iterations (two).
template <int HD, int SG>
union FusedStatLds {
  attn::AttnLds<HD, 1> attn;
  uint32_t pre[SG > 0 ? 2 * 4 * SG * 256 : 4];
};

// Decode passes over contexts of one attention chunk: the QKV GEMM, the
// attention that reads its output and (OKI > 0) the O-projection of the
// attention output in one launch.  Workgroups [0, n_tiles) are GEMM tiles
// (wavefronts 0-3 compute, 4-7 only take part in the workgroup's barriers);
// each stores its Q / K / V at device scope, waits for its stores, and counts
// itself in.  The next n_cons workgroups are the attention workgroups of
// k_attn's single-chunk plan (KV head, query group, sequence): the first pair
// of key tiles, when it precedes the pass, is requested before they wait for
// every GEMM tile; Q and the keys of the pass are then read at device scope.
// With O units their output is stored at device scope and they count
// themselves in; O-projection workers (the QKV workgroups once their tile is
// done, and o_extra workgroups after the attention ones) request their
// weights, wait for every attention workgroup and finish their units
// (o_part).  The counters: FuseCtl.  All workgroups of the launch are
// co-resident (the host checks the grid against the device's occupancy), a
// phase waits only for earlier phases, and every wait is bounded
// (attn::fuse_wait_on), so every wait ends.
template <int MT, int S, int HD, int OKI, int SG, int SD>
__global__ __launch_bounds__(512) void k_qkv_attn(const GemmArgs g, const AttnArgs a, const FuseCtl f,
                                                  const GemmArgs o, const GemmArgs gu, const GemmArgs dn) {
  static_assert(SG == 0 || (MT == 1 && OKI > 0), "gate/up joins only launches with O units");
  static_assert(SD == 0 || (SD == 1 && SG > 0), "the down projection joins only launches with gate/up");
  // [0, gu_lds): reductions (GEMM tiles [4][S * MT * 256], O units [8][2][256],
  // down tiles [4][256]); from gu_lds: preloaded gate/up weights, whose first
  // block of each wavefront later holds that wavefront's gate/up partial tile
  extern __shared__ float red[];
  __shared__ FusedStatLds<HD, SG> stat_sm;
  attn::AttnLds<HD, 1>& attn_sm = stat_sm.attn;
  const int tid = threadIdx.x;
  const int b = blockIdx.x;
  uint32_t* pre_lds = reinterpret_cast<uint32_t*>(reinterpret_cast<char*>(red) + f.gu_lds);
  uint32_t* stat_lds = stat_sm.pre;
  const bool gu_tile = SG > 0 && b < f.gu_tiles;          // uniform
  const int pre = b < g.n_tiles ? f.gu_pre_q : f.gu_pre;
  const int pre_d = pre - min(pre, f.gu_stat);            // the rest go into stat_sm
  auto preload = [&]() {
    if constexpr (SG > 0) {
      if (gu_tile && tid < 256) gu_preload<SG, true>(gu, b, 0, pre, pre, pre_d, pre_lds, stat_lds);
    }
  };
  if (b < g.n_tiles) {
    if (tid < 256) {
      gemm_tile<MT, S, EPI_QKV, true>(g, b, 0, 1, 4, red);
      __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);      // this wavefront's stores are complete
    } else {
      __syncthreads();                              // the tile's reduction barrier
    }
    __syncthreads();
    if (tid == 0)
      __hip_atomic_fetch_add(f.counters + (b % kFuseLanes) * kFuseStride, 1, __ATOMIC_RELAXED,
                             __HIP_MEMORY_SCOPE_AGENT);
    if constexpr (OKI > 0) o_part<OKI, (SG > 0)>(o, f, f.o_extra + b, red, preload);
  } else if (b - g.n_tiles < f.n_cons) {
    const int i = b - g.n_tiles;
    const int kvh = i % a.n_kv, qg = (i / a.n_kv) % a.n_qblocks;
    const unsigned z = i / (a.n_kv * a.n_qblocks);
    attn::attn_tile<HD, 1, 2 * kAttnWaves, true>(a, kvh, qg, z, f, attn_sm);
    if constexpr (OKI > 0) {
      __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);      // this wavefront's output stores are complete
      __syncthreads();
      if (tid < kFuseLanes)   // every counter: each poller reads the one of its XCD
        __hip_atomic_fetch_add(f.counters + (kFuseLanes + tid) * kFuseStride, 1, __ATOMIC_RELAXED,
                               __HIP_MEMORY_SCOPE_AGENT);
    }
    // the gate/up preload only now: issued earlier it competes with the QKV
    // weights that the attention waits for (SG > 0 implies OKI > 0: the
    // barrier above ended the attention's use of stat_sm)
    if constexpr (SG > 0) {
      if (gu_tile && tid < 256) gu_preload<SG, true>(gu, b, 0, pre, pre, pre_d, pre_lds, stat_lds);
    }
  } else {
    if constexpr (OKI > 0) o_part<OKI, (SG > 0)>(o, f, b - g.n_tiles - f.n_cons, red, preload);
  }
  if constexpr (SG > 0) {
    if (gu_tile) {
      __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);      // this wavefront's preloaded weights are in LDS
      if (tid < 256) {
        // the tile's reduction in each wavefront's own first block of the
        // dynamic preload area (read only by that wavefront, before it)
        gemm_tile<1, SG, EPI_SWIGLU, false, 1>(gu, b, 0, 1, 4, reinterpret_cast<float*>(pre_lds), &f, pre_lds, pre,
                                               stat_lds, pre_d, max(pre_d, 1) * SG * 256);
      } else {                                      // the tile's two barriers
        attn::fuse_wait_on<kFuseLanes>(f.counters + 2 * kFuseLanes * kFuseStride, f.n_odone, f.err);
        __syncthreads();
      }
      if constexpr (SD > 0) {                       // h of this tile complete: count in
        __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
        __syncthreads();
        if (tid == 0)
          __hip_atomic_fetch_add(f.counters + (3 * kFuseLanes + b % kFuseLanes) * kFuseStride, 1, __ATOMIC_RELAXED,
                                 __HIP_MEMORY_SCOPE_AGENT);
      }
    }
  }
  if constexpr (SD > 0) {
    if (b < f.d_tiles) {                            // uniform: unit b = (strip, input range)
      const int P = dn.ksplit;
      if (tid < 256) {
        gemm_tile<1, 1, EPI_RESID, false, 2>(dn, b / P, b % P, P, 4, red, &f);
      } else {                                      // the tile's barriers
        attn::fuse_wait_on<kFuseLanes>(f.counters + 3 * kFuseLanes * kFuseStride, f.gu_tiles, f.err);
        __syncthreads();
        if (P > 1) {                                // the partial-tile exchange's two
          __syncthreads();
          __syncthreads();
        }
      }
    }
  }
}

__device__ void commit_verify(const TailArgs& p, const PassSeq& ps, int a, int bonus, const int* res);

// Decode-state update of one sequence once the argmax of its lm rows is
// known (one thread).  Draft: store the candidates, commit only the real rows
// (the mask rows are never committed).  Vanilla draft pass (one of K per
// step, eq. 3): one more candidate, every row committed.  Verify: longest
// agreeing prefix a (eq. 2), bonus t_a, L_t += a + 1, emit the a + 1 tokens;
// in vanilla mode the draft cache keeps the candidates that agree.
__device__ void seq_tail(const TailArgs& p, const PassSeq& ps, const int* res) {
  SeqState* s = p.states + ps.slot;
  if (p.tail == TAIL_PREFILL) {
    s->bonus = res[0];
    s->t[0] = res[0];
    s->pending[0] = res[0];
    s->n_pending = 1;
  } else if (p.tail == TAIL_DRAFT) {
    const int k = s->k;
    for (int i = 0; i < k; ++i) s->cand[i] = res[i];
    s->L[1] = ps.pos0 + ps.n_real;
  } else if (p.tail == TAIL_VSD_DRAFT) {
    s->cand[s->j] = res[0];
    ++s->j;
    s->L[1] = ps.pos0 + ps.n_real;
  } else if (p.tail == TAIL_VERIFY) {
    const int k = s->k;
    int a = 0;
    while (a < k && s->cand[a] == res[a]) ++a;      // longest agreeing prefix
    commit_verify(p, ps, a, res[a], res);
  }
}

// Verify step of one sequence with a accepted candidates and the step's last
// token (greedy: the target's argmax t_a; sampling: the residual or bonus
// draw): L_t += a + 1, emit c_1..c_a and the last token, count the step.
__device__ void commit_verify(const TailArgs& p, const PassSeq& ps, int a, int bonus, const int* res) {
  SeqState* s = p.states + ps.slot;
  {
    const int k = s->k;
    for (int i = 0; i <= k; ++i) s->t[i] = res[i];
    s->a = a;
    s->bonus = bonus;
    s->L[0] = ps.pos0 + a + 1;                     // keep pending + accepted rows
    if (s->vsd && k > 0) {
      // the draft cache holds the pending token and c_1..c_{k-1}; it keeps
      // those that agree, and the tokens after them become pending
      const int keep = min(a, k - 1);
      s->L[1] = ps.pos0 + 1 + keep;
      int n = 0;
      for (int i = keep; i < a; ++i) s->pending[n++] = s->cand[i];
      s->pending[n++] = bonus;
      s->n_pending = n;
      s->j = 0;
    } else {
      for (int i = 0; i < a; ++i) s->pending[i] = s->cand[i];
      s->pending[a] = bonus;
      s->n_pending = a + 1;
    }
    if (p.out_tokens) {                             // emitted: c_1..c_a, then the bonus
      int* out = p.out_tokens + (size_t)ps.slot * p.out_cap;
      for (int i = 0; i <= a; ++i) {
        if (s->n_out < p.out_cap) out[s->n_out] = i < a ? s->cand[i] : bonus;
        ++s->n_out;
      }
    }
    ++s->steps;
    ++s->draw;
    ++s->accept_hist[a];
  }
}

// Rows of one sequence in the pass that follows
//   a draft pass (PARD), or the last vanilla draft pass of a step: the verify
//     pass, [pending, c_1..c_k] at L_t;
//   an earlier vanilla draft pass: the next one, the candidate just drafted;
//   a verify pass with k > 0: the next draft pass, the pending tokens at L_d
//     followed (PARD) by k-1 mask rows, lm rows from the last pending row on;
//   a verify pass with k = 0: the next plain target step.
__device__ bool to_verify(int after, const SeqState& s) {
  return after == TAIL_DRAFT || (after == TAIL_VSD_DRAFT && s.j >= s.k);
}

__device__ void next_rows(int after, const SeqState& s, int* n_rows, int* n_real, int* pos0, int* lm_first,
                          int* lm_rows) {
  const int k = s.k;
  if (to_verify(after, s)) {
    *n_rows = k + 1; *n_real = k + 1; *pos0 = s.L[0]; *lm_first = 0; *lm_rows = k + 1;
  } else if (after == TAIL_VSD_DRAFT) {
    *n_rows = 1; *n_real = 1; *pos0 = s.L[1]; *lm_first = 0; *lm_rows = 1;
  } else if (k > 0 && s.vsd) {
    *n_rows = s.n_pending; *n_real = s.n_pending; *pos0 = s.L[1]; *lm_first = s.n_pending - 1; *lm_rows = 1;
  } else if (k > 0) {
    *n_rows = s.n_pending + k - 1; *n_real = s.n_pending; *pos0 = s.L[1]; *lm_first = s.n_pending - 1; *lm_rows = k;
  } else {
    *n_rows = 1; *n_real = 1; *pos0 = s.L[0]; *lm_first = 0; *lm_rows = 1;
  }
}

__device__ int next_id(int after, const SeqState& s, int i) {
  if (to_verify(after, s)) return i == 0 ? s.bonus : s.cand[i - 1];
  if (after == TAIL_VSD_DRAFT) return s.cand[s.j - 1];
  if (s.k > 0) return i < s.n_pending ? s.pending[i] : s.mask_id;
  return s.bonus;
}

// Stages the next pass of the step for the sequences of the current pass, in
// the same order (run by a whole workgroup).  With drop_done, sequences that
// have written all requested tokens leave the batch.  The current pass's
// sequence list is read before anything is written, so the next descriptor
// may be the current one (plain target steps).
__device__ void stage_next(const TailArgs& p, bool drop_done) {
  __shared__ int sl[kMaxPassSeqs], r0[kMaxPassSeqs + 1], l0[kMaxPassSeqs + 1];
  __shared__ int n_next_s;
  const int tid = threadIdx.x, nth = blockDim.x;
  const int after = p.tail;
  if (tid == 0) {
    const int n_cur = p.desc->n_seq;
    int n = 0, rows = 0, lm = 0;
    for (int j = 0; j < n_cur; ++j) {
      const int slot = p.desc->seq[j].slot;
      const SeqState& s = p.states[slot];
      if (drop_done && after == TAIL_VERIFY && s.n_out >= s.n_target) {
        // its logits are overwritten by the passes that follow without it
        p.lm_map[slot] = int2{0, 0};
        if (p.lm_map_draft) p.lm_map_draft[slot] = int2{0, 0};
        continue;
      }
      int nr, nreal, pos0, lmf, lmr;
      next_rows(after, s, &nr, &nreal, &pos0, &lmf, &lmr);
      sl[n] = slot;
      r0[n] = rows;
      l0[n] = lm;
      rows += nr;
      lm += lmr;
      ++n;
    }
    r0[n] = rows;
    l0[n] = lm;
    n_next_s = n;
  }
  __syncthreads();
  const int n = n_next_s;
  FwdDesc* nd = p.next_desc;
  for (int j = tid; j < n; j += nth) {
    const SeqState& s = p.states[sl[j]];
    PassSeq q{};
    int lmf;
    next_rows(after, s, &q.n_rows, &q.n_real, &q.pos0, &lmf, &q.lm_rows);
    q.slot = sl[j];
    q.row0 = r0[j];
    q.lm0 = l0[j];
    nd->seq[j] = q;
  }
  // rows and lm rows: a thread finds its sequence by binary search over the
  // row offsets
  for (int r = tid; r < r0[n]; r += nth) {
    int lo = 0, hi = n - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (r0[mid] <= r) lo = mid; else hi = mid - 1;
    }
    const SeqState& s = p.states[sl[lo]];
    int nr, nreal, pos0, lmf, lmr;
    next_rows(after, s, &nr, &nreal, &pos0, &lmf, &lmr);
    const int i = r - r0[lo];
    nd->ids[r] = next_id(after, s, i);
    nd->pos[r] = pos0 + i;
    nd->slot[r] = sl[lo];
    if (i >= lmf && i < lmf + lmr) nd->lm_src[l0[lo] + i - lmf] = r;
  }
  if (tid == 0) {
    nd->n_rows = r0[n];
    nd->n_seq = n;
    nd->n_lm = l0[n];
  }
}

// Second argmax pass and step tail.  Workgroup j serves sequence j of the
// pass: wave w reduces its lm rows w, w+16, ... over the tiles, 16
// independent loads per lane in flight at a time; then one thread updates
// the sequence's decode state.  A single-sequence pass also stages the next
// pass here; batched passes stage it in k_stage.
// ---- speculative sampling (temperature T; samp_k = log2(e) / T) ----
// A row's distribution is softmax(z / T).  The LM GEMM left, per tile of
// tile_w columns, the tile's max m_t and s_t = sum 2^((z - m_t) k); the row's
// max M and normaliser S = sum_t s_t 2^((m_t - M) k) follow.  A token is
// drawn by inverse CDF in token-id order: the smallest x whose cumulative
// weight exceeds u S.  All sums run in a fixed order.

__device__ __forceinline__ float tile_weight(float m, float s, float M, float k) {
  return m == -INFINITY ? 0.f : s * __builtin_amdgcn_exp2f((m - M) * k);
}

constexpr int kScanBatch = 8;       // blocks of 64 tiles whose loads are in flight together
constexpr int kResidBlock = 256;    // vocabulary entries per wavefront block of the residual draw (4 per lane)
constexpr int kMaxResidBlocks = kMaxSampleVocab / kResidBlock;

// Tile weights of blocks b0 .. b0 + kScanBatch*64 of lm row lmr, lane-strided (coalesced).
__device__ __forceinline__ void tile_block_weights(const TailArgs& p, int lmr, int b0, float M, int lane,
                                                   float (&w)[kScanBatch]) {
  const float* mv = p.amax_val + (size_t)lmr * p.n_tiles;
  const float* sv = p.amax_sum + (size_t)lmr * p.n_tiles;
#pragma unroll
  for (int u = 0; u < kScanBatch; ++u) {
    const int t = b0 + 64 * u + lane;
    w[u] = t < p.n_tiles ? tile_weight(mv[t], sv[t], M, p.samp_k) : 0.f;
  }
}

// (M, S) of lm row `lmr` (one wavefront): S adds the blocks' sums in block order.
__device__ void row_stats(const TailArgs& p, int lmr, int lane, float* M, float* S) {
  const float* mv = p.amax_val + (size_t)lmr * p.n_tiles;
  float m = -INFINITY;
  for (int t = lane; t < p.n_tiles; t += 64) m = fmaxf(m, mv[t]);
  m = wave_max(m);
  float acc = 0.f;
  for (int b0 = 0; b0 < p.n_tiles; b0 += 64 * kScanBatch) {
    float w[kScanBatch];
    tile_block_weights(p, lmr, b0, m, lane, w);
#pragma unroll
    for (int u = 0; u < kScanBatch; ++u) acc += wave_sum(w[u]);
  }
  *M = m;
  *S = acc;
}

// Draw from lm row `lmr` with uniform u (one wavefront; every lane returns the
// token): the block of 64 tiles where the running sum (the same block sums in
// the same order as S) passes u S, the tile inside it, then the column.
__device__ int wave_sample(const TailArgs& p, int lmr, float M, float S, float u, int lane) {
  const float k = p.samp_k, target = u * S;
  float carry = 0.f, rem = 0.f;
  int tsel = -1;
  for (int b0 = 0; b0 < p.n_tiles && tsel < 0; b0 += 64 * kScanBatch) {
    float w[kScanBatch];
    tile_block_weights(p, lmr, b0, M, lane, w);
#pragma unroll
    for (int v = 0; v < kScanBatch; ++v) {
      if (tsel >= 0) break;                          // uniform
      const float tot = wave_sum(w[v]);
      if (carry + tot > target) {                    // uniform
        const float incl = wave_incl_scan(w[v], lane);
        const uint64_t hit = __ballot(w[v] > 0.f && carry + incl > target);
        const uint64_t nz = __ballot(w[v] > 0.f);
        const int l = hit ? __ffsll((unsigned long long)hit) - 1 : 63 - __clzll((long long)nz);
        tsel = b0 + 64 * v + l;
        rem = target - (carry + __shfl(incl - w[v], l));
      }
      carry += tot;
    }
  }
  if (tsel < 0) {          // u S rounded up to S: the last tile with weight, its last column
    for (int b = (p.n_tiles - 1) / 64 * 64; b >= 0 && tsel < 0; b -= 64) {
      const int t = b + lane;
      const float w = t < p.n_tiles ? tile_weight(p.amax_val[(size_t)lmr * p.n_tiles + t],
                                                  p.amax_sum[(size_t)lmr * p.n_tiles + t], M, k) : 0.f;
      const uint64_t nz = __ballot(w > 0.f);
      if (nz) tsel = b + 63 - __clzll((long long)nz);
    }
    if (tsel < 0) return 0;
    rem = INFINITY;
  }
  // columns of the chosen tile, 64 at a time (one per lane), running sum in column order
  int x = -1, last = -1;
  float ccarry = 0.f;
  for (int c0 = 0; c0 < p.tile_w && x < 0; c0 += 64) {
    const int col = tsel * p.tile_w + c0 + lane;
    float w = 0.f;
    if (c0 + lane < p.tile_w && col < p.vocab)
      w = __builtin_amdgcn_exp2f((p.logits[(size_t)lmr * p.vocab + col] - M) * k);
    const float cincl = wave_incl_scan(w, lane);
    const uint64_t chit = __ballot(w > 0.f && ccarry + cincl > rem);
    const uint64_t cnz = __ballot(w > 0.f);
    if (chit) x = c0 + __ffsll((unsigned long long)chit) - 1;
    if (cnz) last = c0 + 63 - __clzll((long long)cnz);
    ccarry += __shfl(cincl, 63);
  }
  if (x < 0) x = last < 0 ? 0 : last;   // rounding: the tile's last column with weight
  return tsel * p.tile_w + x;
}

// Residual draw at a rejected position: weights max(0, p(x) - q(x)) over the
// vocabulary, p from the target row zp (M_p, S_p), q from the draft row zq
// (M_q, S_q).  Block g holds entries [256 g, 256 g + 256), 4 per lane; the
// wavefronts take blocks round-robin and keep each block's sum in LDS; wave 0
// then scans the block sums in order and the chosen block inside.  Whole
// workgroup; returns -1 when the residual has no mass (only through rounding).
__device__ int block_sample_residual(const TailArgs& p, const float* zp, float Mp, float Sp, const float* zq,
                                     float Mq, float Sq, float u, float* part_s, int* pick_s) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int V = p.vocab, n_blocks = (V + kResidBlock - 1) / kResidBlock;
  const float k = p.samp_k, ip = 1.0f / Sp, iq = 1.0f / Sq;
  auto resid4 = [&](int g, float (&r)[4]) {      // V is a multiple of 16: a lane's 4 entries are all in range or not
    const int x0 = g * kResidBlock + 4 * lane;
    if (x0 < V) {
      const f32x4 a = *reinterpret_cast<const f32x4*>(zp + x0);
      const f32x4 b = *reinterpret_cast<const f32x4*>(zq + x0);
#pragma unroll
      for (int e = 0; e < 4; ++e)
        r[e] = fmaxf(__builtin_amdgcn_exp2f((a[e] - Mp) * k) * ip - __builtin_amdgcn_exp2f((b[e] - Mq) * k) * iq, 0.f);
    } else {
      r[0] = r[1] = r[2] = r[3] = 0.f;
    }
  };
  for (int g0 = wave; g0 < n_blocks; g0 += 16 * kScanBatch) {
    float r[kScanBatch][4];
#pragma unroll
    for (int v = 0; v < kScanBatch; ++v) {
      const int g = g0 + 16 * v;
      if (g < n_blocks) resid4(g, r[v]);
      else r[v][0] = r[v][1] = r[v][2] = r[v][3] = 0.f;
    }
#pragma unroll
    for (int v = 0; v < kScanBatch; ++v) {
      const float t = wave_sum(((r[v][0] + r[v][1]) + r[v][2]) + r[v][3]);
      const int g = g0 + 16 * v;
      if (lane == 0 && g < n_blocks) part_s[g] = t;
    }
  }
  __syncthreads();
  if (wave == 0) {
    float total = 0.f;
    for (int g0 = 0; g0 < n_blocks; g0 += 64) total += wave_sum(g0 + lane < n_blocks ? part_s[g0 + lane] : 0.f);
    int x_sel = -1;
    if (total > 0.f) {
      const float target = u * total;
      float carry = 0.f, rem = INFINITY;
      int gsel = -1;
      for (int g0 = 0; g0 < n_blocks && gsel < 0; g0 += 64) {
        const float w = g0 + lane < n_blocks ? part_s[g0 + lane] : 0.f;
        const float tot = wave_sum(w);
        if (carry + tot > target) {
          const float incl = wave_incl_scan(w, lane);
          const uint64_t hit = __ballot(w > 0.f && carry + incl > target);
          const uint64_t nz = __ballot(w > 0.f);
          const int l = hit ? __ffsll((unsigned long long)hit) - 1 : 63 - __clzll((long long)nz);
          gsel = g0 + l;
          rem = target - (carry + __shfl(incl - w, l));
        }
        carry += tot;
      }
      if (gsel < 0) {      // u * total rounded up to total: the last block with mass
        for (int g = n_blocks - 1; g >= 0; --g)
          if (part_s[g] > 0.f) { gsel = g; break; }
      }
      if (gsel < 0) gsel = 0;   // not reached: total > 0 means some block has mass
      // inside the block: lane sums in lane order, then the lane's 4 entries
      float r[4];
      resid4(gsel, r);
      const float ls = ((r[0] + r[1]) + r[2]) + r[3];
      const float incl = wave_incl_scan(ls, lane);
      const uint64_t hit = __ballot(ls > 0.f && incl > rem);
      const uint64_t nz = __ballot(ls > 0.f);
      const int l = hit ? __ffsll((unsigned long long)hit) - 1 : (nz ? 63 - __clzll((long long)nz) : 0);
      if (lane == l) {
        float acc = incl - ls;
        int last = -1;
        for (int e = 0; e < 4; ++e) {
          if (r[e] > 0.f) last = e;
          if (x_sel < 0 && hit && r[e] > 0.f && acc + r[e] > rem) x_sel = gsel * kResidBlock + 4 * lane + e;
          acc += r[e];
        }
        if (x_sel < 0) x_sel = gsel * kResidBlock + 4 * lane + (last < 0 ? 0 : last);
        pick_s[0] = x_sel;
      }
      if (!nz && lane == 0) pick_s[0] = -1;
    } else if (lane == 0) {
      pick_s[0] = -1;
    }
  }
  __syncthreads();
  return pick_s[0];
}

// Phase clock of the fused loop (one thread): at the start of a step tail the
// verify phase ends (target pass up to its lm_head); at the end of the tail --
// after the next pass is staged -- the draft phase (draft pass and tail) or the
// accept phase (verify tail) ends, and a verify tail records the step's end.
__device__ void clock_tail_start(const TailArgs& p) {
  if (p.tail != TAIL_VERIFY) return;
  const unsigned long long t = wall_clock64();
  p.clock->tail_start = t;
  p.clock->verify_ticks += t - p.clock->pass_start[0];
}
__device__ void clock_tail_end(const TailArgs& p) {
  const unsigned long long t = wall_clock64();
  PhaseClock* c = p.clock;
  if (p.tail == TAIL_DRAFT || p.tail == TAIL_VSD_DRAFT) {
    c->draft_ticks += t - c->pass_start[1];
  } else if (p.tail == TAIL_VERIFY) {
    c->accept_ticks += t - c->tail_start;
    c->step_end[c->n_steps % kStepRing] = t;
    ++c->n_steps;
  }
}

__global__ __launch_bounds__(1024) void k_lm_tail(const TailArgs p) {
  __shared__ int res_s[kMaxK + 1];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const FwdDesc* dp = p.desc;
  const int sj = blockIdx.x;
  if (sj >= dp->n_seq) return;                    // uniform: the whole block leaves
  // block 0 keeps the clock; with several sequences k_stage (the kernel after
  // this one) ends the phase
  const bool clock = p.clock && blockIdx.x == 0;
  if (clock && tid == 0) clock_tail_start(p);
  const PassSeq ps = dp->seq[sj];
  const int rows = min(ps.lm_rows, kMaxK + 1);
  for (int r = wave; r < rows; r += 16) {
    float bv = -INFINITY;
    int bi = INT_MAX;
    const float* vals = p.amax_val + (size_t)(ps.lm0 + r) * p.n_tiles;
    const int* idxs = p.amax_idx + (size_t)(ps.lm0 + r) * p.n_tiles;
    for (int t0 = lane; t0 < p.n_tiles; t0 += 64 * 16) {
      float xv[16];
      int xi[16];
#pragma unroll
      for (int u = 0; u < 16; ++u) {
        const int t = t0 + 64 * u;
        xv[u] = t < p.n_tiles ? vals[t] : -INFINITY;
        xi[u] = t < p.n_tiles ? idxs[t] : INT_MAX;
      }
#pragma unroll
      for (int u = 0; u < 16; ++u)
        if (better(xv[u], xi[u], bv, bi)) { bv = xv[u]; bi = xi[u]; }
    }
    for (int off = 32; off > 0; off >>= 1) {
      const float ov = __shfl_xor(bv, off);
      const int oi = __shfl_xor(bi, off);
      if (better(ov, oi, bv, bi)) { bv = ov; bi = oi; }
    }
    if (lane == 0) res_s[r] = (bi >= 0 && bi < p.vocab) ? bi : 0;
  }
  const bool sampling =
      p.samp_k > 0.f && (p.tail == TAIL_PREFILL || p.tail == TAIL_DRAFT || p.tail == TAIL_VERIFY);
  if (!sampling) {
    __syncthreads();
    if (tid == 0) {
      for (int r = 0; r < rows; ++r) p.result[ps.lm0 + r] = res_s[r];
      p.lm_map[ps.slot] = int2{ps.lm0, rows};
      seq_tail(p, ps, res_s);
    }
  } else {
    // speculative sampling: draft candidates and the first token are drawn
    // from their rows; a verify pass runs the keep tests in order and draws
    // the step's last token from the residual (first rejection) or from the
    // bonus row (all kept)
    __shared__ float Ms[kMaxK + 1], Ss[kMaxK + 1];
    __shared__ float part_s[kMaxResidBlocks];
    __shared__ int pick_s[2], a_s, tok_s;
    SeqState* st = p.states + ps.slot;
    const int draw = st->draw;
    for (int r = wave; r < rows; r += 16) {
      float M, S;
      row_stats(p, ps.lm0 + r, lane, &M, &S);
      if (lane == 0) { Ms[r] = M; Ss[r] = S; }
    }
    __syncthreads();
    if (p.tail == TAIL_DRAFT || p.tail == TAIL_PREFILL) {
      const int purpose = p.tail == TAIL_PREFILL ? PURPOSE_FIRST : PURPOSE_DRAFT;
      for (int r = wave; r < rows; r += 16) {
        const int x = wave_sample(p, ps.lm0 + r, Ms[r], Ss[r], sample_uniform(p.seed, ps.slot, draw, r, purpose), lane);
        if (lane == 0) res_s[r] = x;
      }
      if (p.tail == TAIL_DRAFT && tid < min(rows, kMaxK)) {   // the draft's rows, for the keep tests
        st->qM[tid] = Ms[tid];
        st->qS[tid] = Ss[tid];
      }
      __syncthreads();
      if (tid == 0) {
        for (int r = 0; r < rows; ++r) p.result[ps.lm0 + r] = res_s[r];
        p.lm_map[ps.slot] = int2{ps.lm0, rows};
        seq_tail(p, ps, res_s);
      }
    } else {   // TAIL_VERIFY
      const int k = st->k;
      if (wave == 0) {
        // keep test of position j in lane j (k <= 32); a = the first position not kept
        const int2 dm = p.lm_map_draft[ps.slot];   // this slot's rows of the draft's last pass
        bool keep = true;
        if (lane < k) {
          const int x = st->cand[lane];
          const float pz = p.logits[(size_t)(ps.lm0 + lane) * p.vocab + x];
          const float qz = p.q_logits[(size_t)(dm.x + lane) * p.vocab + x];
          const float pp = __builtin_amdgcn_exp2f((pz - Ms[lane]) * p.samp_k) / Ss[lane];
          const float qq = __builtin_amdgcn_exp2f((qz - st->qM[lane]) * p.samp_k) / st->qS[lane];
          keep = sample_uniform(p.seed, ps.slot, draw, lane, PURPOSE_KEEP) * qq < pp;
        }
        const uint64_t rejected = __ballot(!keep);
        if (lane == 0) a_s = rejected ? __ffsll((unsigned long long)rejected) - 1 : k;
      }
      __syncthreads();
      const int a = a_s;
      const float u = sample_uniform(p.seed, ps.slot, draw, a, PURPOSE_LAST);
      int tok = -1;
      if (a < k) {
        const int2 dm = p.lm_map_draft[ps.slot];
        tok = block_sample_residual(p, p.logits + (size_t)(ps.lm0 + a) * p.vocab, Ms[a], Ss[a],
                                    p.q_logits + (size_t)(dm.x + a) * p.vocab, st->qM[a], st->qS[a], u, part_s,
                                    pick_s);
      }
      if (tok < 0) {                                // bonus row (or a residual without mass)
        if (wave == 0) {
          const int x = wave_sample(p, ps.lm0 + a, Ms[a], Ss[a], u, lane);
          if (lane == 0) tok_s = x;
        }
      } else if (tid == 0) {
        tok_s = tok;
      }
      __syncthreads();
      if (tid == 0) {
        for (int r = 0; r < rows; ++r) p.result[ps.lm0 + r] = res_s[r];
        p.lm_map[ps.slot] = int2{ps.lm0, rows};
        commit_verify(p, ps, a, tok_s, res_s);
      }
    }
  }
  if (gridDim.x == 1 && p.next_desc) {
    __syncthreads();
    stage_next(p, false);
  }
  if (clock && (gridDim.x == 1 || !p.next_desc)) {
    __syncthreads();
    if (tid == 0) clock_tail_end(p);
  }
}

__global__ __launch_bounds__(256) void k_stage(const TailArgs p) {
  stage_next(p, true);
  if (p.clock) {
    __syncthreads();
    if (threadIdx.x == 0) clock_tail_end(p);
  }
}

// ============================================================================
// Row-block GEMM: passes of more than kMaxRows rows (batched decode passes,
// where the GEMMs are dense contractions at a few hundred rows).
//
// A workgroup of kRowsWaves wavefronts owns kRowTiles*16 (144) rows x 16
// strips (256 columns) over one input range.  The block's rows of A pass
// through LDS one k-block (9 KiB) at a time and are shared by the wavefronts;
// each wavefront streams its own 4 strips of W from HBM straight into the MFMA
// B-operand registers and accumulates 9 x 4 tiles of 16x16 (per k-block:
// 9 KiB of LDS reads and 4 KiB of weights for 36 MFMAs).  The k-blocks are
// software-pipelined (loads 4 k-blocks ahead, A through LDS 2 ahead and into
// fragment registers 1 ahead), so the MFMAs of a k-block wait on nothing
// requested in the same iteration.  Row tiles past the pass's
// rows skip their MFMAs; row blocks past them leave at once.
//
// Blocks are numbered so that the row blocks of one column tile run on the
// same XCD at about the same time (the hardware deals block i to XCD i % 8):
// the later blocks' weight reads then hit that XCD's L2 rather than HBM.
// Narrow GEMMs split the input dimension (ksplit > 1) to fill the chip; each
// split writes an fp32 partial tile and k_gemm_rows_red adds them in split
// order and runs the epilogue, so results are deterministic.
// ============================================================================

typedef f32x4 RowsAcc[kRowTiles][kRowsWaveStrips];

// Compile-time loop: f(integral_constant<int, I>) for I in [B, E).  The row
// tiles of an accumulator are walked this way so that every index is a
// constant whatever the loop body's size: the accumulators then stay in
// registers (a rolled loop would index them dynamically, in scratch memory).
template <int B, int E, class F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (B < E) {
    f(std::integral_constant<int, B>{});
    static_for<B + 1, E>(f);
  }
}

// 1/rms of the block's rows from the producer's per-tile sums of squares
// (fixed order), 16 threads per row.
template <bool LM>
__device__ __forceinline__ void rows_scales(const GemmArgs& p, const FwdDesc* dp, int row0, int row_count, float* rs_s,
                                            int mt_only = -1) {
  // 16 threads per row, rows tid / 16 + 16 k: every row's loads are in flight
  // together (one round of loads per 64 tiles, not one per row), each thread
  // adding its tiles in increasing order.  mt_only >= 0: the rows of that row
  // tile only (rs_s entries of the others are not written).
  const int tid = threadIdx.x;
  constexpr int R = kRowTiles;                     // rows per thread group
  int src[R];
  float t[R];
#pragma unroll
  for (int k = 0; k < R; ++k) {
    const int gr = row0 + (tid >> 4) + 16 * (mt_only >= 0 ? mt_only : k);
    src[k] = gr < row_count ? (LM ? dp->lm_src[gr] : gr) : 0;
    t[k] = 0.f;
  }
  const int n_k = mt_only >= 0 ? 1 : R;            // uniform
  for (int q0 = tid & 15; q0 < p.ss_tiles; q0 += 64) {
    float part[R][4];
#pragma unroll
    for (int k = 0; k < R; ++k)
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const int q = q0 + 16 * u;
        part[k][u] = q < p.ss_tiles && k < n_k ? p.ss_in[(size_t)src[k] * p.ss_stride + q] : 0.f;
      }
#pragma unroll
    for (int k = 0; k < R; ++k)
#pragma unroll
      for (int u = 0; u < 4; ++u) t[k] += part[k][u];
  }
#pragma unroll
  for (int k = 0; k < R; ++k) {
    float v = t[k];
    v += __shfl_xor(v, 8);
    v += __shfl_xor(v, 4);
    v += __shfl_xor(v, 2);
    v += __shfl_xor(v, 1);
    if ((tid & 15) == 0 && k < n_k) rs_s[(tid >> 4) + 16 * (mt_only >= 0 ? mt_only : k)] = 1.0f / sqrtf(v * p.inv_k + p.eps);
  }
}

// Epilogue of one wavefront's accumulators, row tiles [mt_lo, mt_live).  Lane
// l holds, for row tile mt and strip s, column (strip*16 + l%16) of rows
// mt*16 + 4*(l/16) + i.
template <int EPI>
__device__ __forceinline__ void rows_epilogue(const GemmArgs& p, const FwdDesc* dp, RowsAcc& acc, int tile, int row0,
                                              int row_count, int mt_lo, int mt_live, int wave, int lane,
                                              const float* rs_s, u32x4* o_lds = nullptr) {
  const int c16 = lane & 15, g4 = lane >> 4;
  const int strip0 = tile * kRowsTileStrips + wave * kRowsWaveStrips;
  [[maybe_unused]] bool bad = false;
  if constexpr (EPI == EPI_QKV) {
    static_for<0, kRowTiles>([&](auto mtc) __attribute__((always_inline)) {
      constexpr int mt = decltype(mtc)::value;
      if (mt < mt_lo || mt >= mt_live) return;       // uniform
#pragma unroll
      for (int s = 0; s < kRowsWaveStrips; ++s) {
        const int n = (strip0 + s) * 16 + c16;
        const bool col_ok = strip0 + s < p.n_strips;
        const float bias = (col_ok && p.bias) ? p.bias[n] : 0.f;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int rl = mt * 16 + g4 * 4 + i, r = row0 + rl;
          float y = acc[mt][s][i] * rs_s[rl] + bias;
          // rotary partner column (n ^ 1) is in lane l ^ 1 (DPP quad swap)
          const float partner = __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, y), 0xB1,
                                                                                   0xF, 0xF, false));
          if (col_ok && r < row_count) {
            const int pos = dp->pos[r];
            const size_t cache = (size_t)dp->slot[r] * p.kv_seq_stride;
            if (n < p.q_dim + p.kv_dim) {
              const float2 cs = p.rope[(size_t)pos * (p.hd / 2) + ((n % p.hd) >> 1)];
              y = (n & 1) ? (y * cs.x + partner * cs.y) : (y * cs.x - partner * cs.y);
            }
            const uint16_t b = f16_flagged(y, bad);
            if (n < p.q_dim) {
              p.out[(size_t)r * p.ld_out + n] = b;
            } else if (n < p.q_dim + p.kv_dim) {
              const int c = n - p.q_dim;
              p.kc[cache + (size_t)(c / p.hd) * p.cap * p.hd + k_index(pos, c % p.hd, p.hd)] = b;
            } else {
              const int c = n - p.q_dim - p.kv_dim;
              const size_t blk = (size_t)(c / p.hd) * (p.cap / 32) + (pos >> 5);
              p.vc[cache + (blk * p.hd + (c % p.hd)) * 32 + v_slot(pos & 31)] = b;
            }
          }
        }
      }
    });
    flag_range(bad, p.ovf);
  } else if constexpr (EPI == EPI_RESID) {
    float* ss = p.ss_out + (tile * kRowsWaves + wave);
    static_for<0, kRowTiles>([&](auto mtc) __attribute__((always_inline)) {
      constexpr int mt = decltype(mtc)::value;
      if (mt < mt_lo || mt >= mt_live) return;       // uniform
      float sq[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < kRowsWaveStrips; ++s) {
        const int n = (strip0 + s) * 16 + c16;
        if (strip0 + s >= p.n_strips) continue;      // uniform
        const float g = p.g_next[n];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int r = row0 + mt * 16 + g4 * 4 + i;
          if (r < row_count) {
            const size_t o = (size_t)r * p.ldx + n;
            const float xn = p.x[o] + acc[mt][s][i];   // residual + projection
            p.x[o] = xn;
            p.xg[act_index(r, n, p.act_rows)] = f16_flagged(xn * g, bad);
            sq[i] += xn * xn;
          }
        }
      }
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float t = sum16(sq[i]);
        const int r = row0 + mt * 16 + g4 * 4 + i;
        if (c16 == 0 && r < row_count) ss[(size_t)r * p.ss_stride] = t;
      }
    });
    flag_range(bad, p.ovf);
  } else if constexpr (EPI == EPI_SWIGLU) {
    // 8 gate columns then the 8 up columns of the same features per strip.
    // The wavefront's 4 strips are the 32 features of one k-block of h
    // (block tile * 4 + wave): with o_lds (this wavefront's 9 KiB) the block
    // is assembled in LDS and written with 16-byte stores, one row's 64 bytes
    // per 4 lanes (2-byte stores straight from the accumulator layout made the
    // epilogue as long as the GEMM); without, each lane stores its values.
    static_for<0, kRowTiles>([&](auto mtc) __attribute__((always_inline)) {
      constexpr int mt = decltype(mtc)::value;
      if (mt < mt_lo || mt >= mt_live) return;       // uniform
#pragma unroll
      for (int s = 0; s < kRowsWaveStrips; ++s) {
        if (strip0 + s >= p.n_strips) continue;      // uniform
        const int f = (strip0 + s) * 8 + c16;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int rl = mt * 16 + g4 * 4 + i, r = row0 + rl;
          const float gt = acc[mt][s][i] * rs_s[rl];
          // the up value of lane l < 8 is in lane l + 8 of its row of 16 (DPP row rotate by 8)
          const float up = __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, gt), 0x128,
                                                                              0xF, 0xF, false));
          // silu(g) = g / (1 + e^-g), with the hardware exp2 and reciprocal
          const float h = gt * __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(-gt * attn::kLog2e)) * up;
          bool bad_h = false;
          const uint16_t hb = f16_flagged(h, bad_h);
          bad |= bad_h && c16 < 8 && r < row_count;
          if (o_lds) {
            // rows rl, chunk s (features s*8 .. s*8+7): lane pairs pack two
            // values into one dword (DPP quad swap); chunks are swizzled by
            // (rl / 4) % 4 so the four rows of one store land in different banks
            const uint32_t pair =
                (uint32_t)hb | ((uint32_t)__builtin_amdgcn_mov_dpp((int)hb, 0xB1, 0xF, 0xF, false) << 16);
            if (c16 < 8 && !(c16 & 1))
              reinterpret_cast<uint32_t*>(o_lds)[(rl * 4 + (s ^ ((rl >> 2) & 3))) * 4 + (c16 >> 1)] = pair;
          } else if (c16 < 8 && r < row_count) {
            p.out[act_index(r, f, p.act_rows)] = hb;
          }
        }
      }
    });
    if (o_lds) {
      // this wavefront's rows [row0 + 16 mt_lo, row0 + 16 mt_live) of block tile * 4 + wave
      const int blk = tile * kRowsWaves + wave;
      if (blk * 4 < p.n_strips) {                    // uniform: the block holds features of the weight
        for (int e = mt_lo * 64 + lane; e < mt_live * 64; e += 64) {
          const int rl = e >> 2, c = e & 3, r = row0 + rl;
          const u32x4 v = o_lds[rl * 4 + (c ^ ((rl >> 2) & 3))];
          if (r < row_count)
            *reinterpret_cast<u32x4*>(p.out + act_index(r, blk * 32 + c * 8, p.act_rows)) = v;
        }
      }
    }
    flag_range(bad, p.ovf);
  } else {  // EPI_LOGITS
    static_for<0, kRowTiles>([&](auto mtc) __attribute__((always_inline)) {
      constexpr int mt = decltype(mtc)::value;
      if (mt < mt_lo || mt >= mt_live) return;       // uniform
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int rl = mt * 16 + g4 * 4 + i, r = row0 + rl;
        float bv = -INFINITY;
        int bi = INT_MAX;
#pragma unroll
        for (int s = 0; s < kRowsWaveStrips; ++s) {
          const int n = (strip0 + s) * 16 + c16;
          if (strip0 + s >= p.n_strips) continue;    // uniform
          const float val = acc[mt][s][i] * rs_s[rl];
          if (r < row_count) p.logits[(size_t)r * p.vocab + n] = val;
          if (better(val, n, bv, bi)) { bv = val; bi = n; }
        }
#pragma unroll
        for (int off = 8; off > 0; off >>= 1) {
          const float ov = __shfl_xor(bv, off);
          const int oi = __shfl_xor(bi, off);
          if (better(ov, oi, bv, bi)) { bv = ov; bi = oi; }
        }
        if (c16 == 0 && r < row_count) {
          p.amax_val[(size_t)r * p.amax_stride + tile * kRowsWaves + wave] = bv;
          p.amax_idx[(size_t)r * p.amax_stride + tile * kRowsWaves + wave] = bi;
        }
        if (p.samp_k > 0.f) {       // sampling: the entry's softmax weight relative to its max
          float sw = 0.f;
#pragma unroll
          for (int s = 0; s < kRowsWaveStrips; ++s) {
            if (strip0 + s >= p.n_strips) continue;  // uniform
            sw += __builtin_amdgcn_exp2f((acc[mt][s][i] * rs_s[rl] - bv) * p.samp_k);
          }
#pragma unroll
          for (int off = 8; off > 0; off >>= 1) sw += __shfl_xor(sw, off);
          if (c16 == 0 && r < row_count) p.amax_sum[(size_t)r * p.amax_stride + tile * kRowsWaves + wave] = sw;
        }
      }
    });
  }
}

// Block id -> (column tile, input split, row block), row blocks fastest and
// consecutive ids on one XCD.
__device__ __forceinline__ void rows_block(const GemmArgs& p, int* tile, int* ks, int* mb) {
  const int G = gridDim.x, bid = blockIdx.x;
  const int per = G / 8, rem = G % 8, xcd = bid % 8, slot = bid / 8;
  const int lid = xcd * per + min(xcd, rem) + slot;
  *mb = lid % p.m_blocks;
  const int rest = lid / p.m_blocks;
  *ks = rest % p.ksplit;
  *tile = rest / p.ksplit;
}

template <int EPI>
__global__ __launch_bounds__(256) void k_gemm_rows(const GemmArgs p) {
  constexpr int MB = kRowTiles, NS = kRowsWaveStrips;
  constexpr int AE = MB * 64;                        // 16-byte A elements of one k-block
  constexpr int AJ = (AE + 255) / 256;               // per thread
  constexpr bool LM = EPI == EPI_LOGITS;             // rows are the pass's lm rows
  // (padded to whole rounds of the workgroup's threads: every thread stores
  // each of its AJ elements, those past AE are zeros never read)
  __shared__ __attribute__((aligned(16))) u32x4 a_lds[2][AJ * 256];
  // SwiGLU: each wavefront's block of h (MB * 16 rows x 64 bytes) for 16-byte stores
  __shared__ __attribute__((aligned(16))) u32x4 o_lds[EPI == EPI_SWIGLU ? kRowsWaves * MB * 64 : 1];
  __shared__ float rs_s[MB * 16];

  int tile, ks, mb;
  rows_block(p, &tile, &ks, &mb);
  const FwdDesc* dp = p.desc;
  const int row_count = LM ? dp->n_lm : dp->n_rows;
  const int row0 = mb * MB * 16;
  if (row0 >= row_count) return;                     // uniform: the whole block leaves
  const int mt_live = min(MB, (row_count - row0 + 15) / 16);
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int kb0 = ks * p.kb_total / p.ksplit, kb1 = (ks + 1) * p.kb_total / p.ksplit;
  const int n_kb = kb1 - kb0;

  // W: this wavefront's strips, block (kb, strip) at (kb * n_strips + strip) KiB
  const int strip0 = tile * kRowsTileStrips + wave * NS;
  const __amdgpu_buffer_rsrc_t wrs = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(p.W), 0, (int)min((size_t)p.n_strips * p.kb_total * 1024, (size_t)0x7fffffff),
      kRsrcWord3);
  // strips past the weight's last one (only in the last column tile) read
  // zeros or neighbouring weights: their columns are never stored
  const int w_voff = (strip0 * 64 + lane) * 16;

  // A: element e of a k-block is 16 bytes of block row e / 4; rows past the
  // pass read as zeros (offset beyond the buffer)
  const __amdgpu_buffer_rsrc_t ars = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(p.A), 0, p.act_rows * p.lda * 2, kRsrcWord3);
  constexpr int kOutOfRange = 0x7FFFFFF0;
  int a_voff[AJ];
#pragma unroll
  for (int j = 0; j < AJ; ++j) {
    const int e = tid + 256 * j;
    const int gr = row0 + (e >> 2);
    const int src = gr < row_count ? (LM ? dp->lm_src[gr] : gr) : 0;
    a_voff[j] = (e < AE && gr < row_count) ? src * 64 + (e & 3) * 16 : kOutOfRange;
  }

  // Software pipeline over the k-blocks.  k-block k's weights are loaded into
  // a register ring D = 4 k-blocks ahead; its A rows are loaded into registers
  // 6 k-blocks ahead, written to LDS (one of two buffers) 2 ahead and read
  // into fragment registers 1 ahead, so each iteration's MFMAs wait on
  // nothing issued in the last few iterations: iteration it reads A(it + 1)'s
  // fragments and writes A(it + 2) to LDS, multiplies k-block it, then
  // requests A(it + 6) and W(it + 4).  One barrier per k-block separates an
  // LDS buffer's writes from its reads.  Indices past the range are clamped
  // (cache hits, never multiplied), so every iteration issues the same loads
  // on every path, in the same order (the compiler's waits then hold the
  // intended depth).
  constexpr int D = 4, DA = 4;   // weight ring, A register ring (A is requested 6 k-blocks ahead)
  static_assert(D % DA == 0 && DA % 2 == 0, "one unrolled turn of the weight ring turns the others whole");
  u32x4 wr[D][NS], ar[DA][AJ], av[2][MB];
  auto issue_a = [&](int slot, int it) {
    const int kb = kb0 + min(it, n_kb - 1);
#pragma unroll
    for (int j = 0; j < AJ; ++j)
      ar[slot][j] = __builtin_amdgcn_raw_buffer_load_b128(ars, a_voff[j], kb * (p.act_rows * 64), 0);
  };
  // LDS holds row r's 16-byte chunk c at r * 4 + (c ^ ((r >> 1) & 3)): a
  // fragment read (lanes 0-15 take rows 0-15 of one chunk) then touches
  // eight different 16-byte bank groups per eight lanes instead of two
  auto swz = [](int e) { return (e & ~3) | ((e & 3) ^ ((e >> 3) & 3)); };
  auto put_a = [&](int slot, int buf) {
#pragma unroll
    for (int j = 0; j < AJ; ++j) a_lds[buf][swz(tid + 256 * j)] = ar[slot][j];
  };
  auto read_a = [&](int slot, int buf) {
#pragma unroll
    for (int mt = 0; mt < MB; ++mt) av[slot][mt] = a_lds[buf][swz((mt * 16 + (lane & 15)) * 4 + (lane >> 4))];
  };

  RowsAcc acc;
#pragma unroll
  for (int mt = 0; mt < MB; ++mt)
#pragma unroll
    for (int s = 0; s < NS; ++s) acc[mt][s] = f32x4{0.f, 0.f, 0.f, 0.f};

  // one strip's MFMAs (row tiles past the pass multiply zeros: no branches
  // between the fragment reads and the MFMAs)
  auto mma_strip = [&](int wslot, int aslot, int s) {
#pragma unroll
    for (int mt = 0; mt < MB; ++mt)
      acc[mt][s] = __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8, av[aslot][mt]),
                                                          __builtin_bit_cast(f16x8, wr[wslot][s]), acc[mt][s], 0, 0, 0);
  };
  auto issue_w_strip = [&](int slot, int it, int s) {
    const int kb = kb0 + min(it, n_kb - 1);
    wr[slot][s] = __builtin_amdgcn_raw_buffer_load_b128(wrs, w_voff, (kb * p.n_strips + s) * 1024, kCachePolicyNT);
  };
  // the A fragments of row tiles [m0, m1)
  auto read_a_part = [&](int slot, int buf, int m0, int m1) {
#pragma unroll
    for (int mt = m0; mt < m1; ++mt) av[slot][mt] = a_lds[buf][swz((mt * 16 + (lane & 15)) * 4 + (lane >> 4))];
  };

  if (n_kb > 0) {
    // A(0) and A(1) into LDS, then the loads of the four turns before the
    // first in the loop's order (W(k + 4) strip 0, A(k + 6), W(k + 4) strips
    // 1-3, for k = -4 .. -1), so the waits the compiler places at the loop's
    // top match every turn's
    issue_a(0, 0);
    issue_a(1, 1);
    __builtin_amdgcn_sched_barrier(0);
    put_a(0, 0);
    put_a(1, 1);
#pragma unroll
    for (int k = -D; k < 0; ++k) {
#pragma unroll
      for (int s2 = 0; s2 < NS; ++s2) {
        __builtin_amdgcn_sched_barrier(0);
        if (s2 == 1 && k >= -4) issue_a((k + 6) % DA, k + 6);   // A(2) .. A(5)
        issue_w_strip(k + D, k + D, s2);
      }
    }
    __builtin_amdgcn_sched_barrier(0);
    __syncthreads();
    read_a(0, 0);
    __syncthreads();                                 // buffer 0 is free again
    // One wavefront issues its loads and LDS operations in order with its
    // MFMAs, so they are interleaved: after each strip's MFMAs go that strip's
    // next weight load (its registers are free then) and a share of the
    // fragment reads of A(it + 1); A(it + 2) goes to LDS after the first strip
    // and A(it + 6) is requested after the second.  The issue cost of the
    // loads and LDS operations then hides under the MFMAs in flight (issued
    // as blocks they measured ~650 cycles per k-block against ~650 of MFMA).
    const int n_it = (n_kb + D - 1) / D * D;
    for (int it0 = 0; it0 < n_it; it0 += D) {
#pragma unroll
      for (int d = 0; d < D; ++d) {
        const int it = it0 + d;
#pragma unroll
        for (int s = 0; s < NS; ++s) {
          if (it < n_kb) mma_strip(d, d & 1, s);     // uniform
          __builtin_amdgcn_sched_barrier(0);
          if (s == 1) issue_a((d + 2) % DA, it + 6);
          issue_w_strip(d, it + D, s);
          __builtin_amdgcn_sched_barrier(0);
          // A(it + 1): written before the last barrier; row tiles 3s .. 3s + 2
          read_a_part((d + 1) & 1, (d + 1) & 1, min(3 * s, MB), min(3 * s + 3, MB));
          if (s == 0) put_a((d + 2) % DA, d & 1);    // A(it + 2) into A(it)'s buffer
          __builtin_amdgcn_sched_barrier(0);
        }
        __syncthreads();
      }
    }
  }

  if (p.ksplit > 1) {
    // partial tile of this split, in register order (coalesced)
    float* part = p.part + ((size_t)(tile * p.m_blocks + mb) * p.ksplit + ks) * kRowsPartFloats;
    static_for<0, MB>([&](auto mtc) __attribute__((always_inline)) {
      constexpr int mt = decltype(mtc)::value;
      if (mt >= mt_live) return;                     // uniform
#pragma unroll
      for (int s = 0; s < NS; ++s)
        *reinterpret_cast<f32x4*>(part + (((wave * MB + mt) * NS + s) * 64 + lane) * 4) = acc[mt][s];
    });
    return;
  }
  if constexpr (EPI != EPI_RESID) {
    rows_scales<LM>(p, dp, row0, row_count, rs_s);
    __syncthreads();
  }
  rows_epilogue<EPI>(p, dp, acc, tile, row0, row_count, 0, mt_live, wave, lane, rs_s,
                    EPI == EPI_SWIGLU ? o_lds + wave * MB * 64 : nullptr);
}

// Sum of the input splits of k_gemm_rows in split order, then the epilogue.
// One workgroup per 16-row tile of a row block (wavefront w takes GEMM
// wavefront w's columns); each thread has the loads of up to 8 splits in
// flight at a time.
template <int EPI>
__global__ __launch_bounds__(256) void k_gemm_rows_red(const GemmArgs p) {
  constexpr int MB = kRowTiles, NS = kRowsWaveStrips;
  constexpr bool LM = EPI == EPI_LOGITS;
  __shared__ float rs_s[MB * 16];
  const int mt_sel = blockIdx.x % MB;
  const int tile = blockIdx.x / (MB * p.m_blocks), mb = (blockIdx.x / MB) % p.m_blocks;
  const FwdDesc* dp = p.desc;
  const int row_count = LM ? dp->n_lm : dp->n_rows;
  const int row0 = mb * MB * 16;
  if (row0 + mt_sel * 16 >= row_count) return;      // uniform
  const int mt_live = min(MB, (row_count - row0 + 15) / 16);
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  if constexpr (EPI != EPI_RESID) rows_scales<LM>(p, dp, row0, row_count, rs_s, mt_sel);
  const float* base = p.part + (size_t)(tile * p.m_blocks + mb) * p.ksplit * kRowsPartFloats +
                      (size_t)(((wave * MB + mt_sel) * NS) * 64 + lane) * 4;
  f32x4 sum[NS];
#pragma unroll
  for (int s = 0; s < NS; ++s) sum[s] = f32x4{0.f, 0.f, 0.f, 0.f};
  for (int k0 = 0; k0 < p.ksplit; k0 += 8) {
    f32x4 v[8][NS];
#pragma unroll
    for (int u = 0; u < 8; ++u)
#pragma unroll
      for (int s = 0; s < NS; ++s)
        v[u][s] = k0 + u < p.ksplit ? *reinterpret_cast<const f32x4*>(base + (size_t)(k0 + u) * kRowsPartFloats + s * 256)
                                    : f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int u = 0; u < 8; ++u)
#pragma unroll
      for (int s = 0; s < NS; ++s)
        if (k0 + u < p.ksplit) sum[s] += v[u][s];
  }
  RowsAcc acc;
  static_for<0, MB>([&](auto mtc) __attribute__((always_inline)) {
    constexpr int mt = decltype(mtc)::value;
#pragma unroll
    for (int s = 0; s < NS; ++s) acc[mt][s] = mt == mt_sel ? sum[s] : f32x4{0.f, 0.f, 0.f, 0.f};
  });
  if constexpr (EPI != EPI_RESID) __syncthreads();
  rows_epilogue<EPI>(p, dp, acc, tile, row0, row_count, mt_sel, min(mt_live, mt_sel + 1), wave, lane, rs_s);
}

template <int EPI>
hipError_t launch_rows(const GemmArgs& a, hipStream_t st, LaunchEvents ev) {
  const int grid = a.n_tiles * a.m_blocks * a.ksplit;
  if (ev.start) {
    hipExtLaunchKernelGGL(k_gemm_rows<EPI>, dim3(grid), dim3(256), 0u, st, ev.start, a.ksplit > 1 ? nullptr : ev.stop,
                          0u, a);
  } else {
    k_gemm_rows<EPI><<<grid, 256, 0, st>>>(a);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || a.ksplit == 1) return e;
  if (ev.start) {
    hipExtLaunchKernelGGL(k_gemm_rows_red<EPI>, dim3(a.n_tiles * a.m_blocks * kRowTiles), dim3(256), 0u, st, nullptr, ev.stop,
                          0u, a);
  } else {
    k_gemm_rows_red<EPI><<<a.n_tiles * a.m_blocks * kRowTiles, 256, 0, st>>>(a);
  }
  return hipGetLastError();
}

template <int EPI, int MT, int S>
hipError_t launch_one(int nw, const GemmArgs& a, hipStream_t st, LaunchEvents ev) {
  const size_t lds = (size_t)nw * S * MT * 256 * sizeof(float);
  if (nw > 8) return hipErrorInvalidValue;
  if (ev.start) {
    hipExtLaunchKernelGGL(k_gemm<MT, S, EPI>, dim3(a.n_tiles, a.ksplit), dim3(64 * nw), (uint32_t)lds, st, ev.start, ev.stop,
                          0u, a);
  } else {
    k_gemm<MT, S, EPI><<<dim3(a.n_tiles, a.ksplit), dim3(64 * nw), lds, st>>>(a);
  }
  return hipGetLastError();
}

template <int EPI, int MT>
hipError_t launch_s(int S, int nw, const GemmArgs& a, hipStream_t st, LaunchEvents ev) {
  switch (S) {
    case 1: return launch_one<EPI, MT, 1>(nw, a, st, ev);
    case 2: return launch_one<EPI, MT, 2>(nw, a, st, ev);
    case 4: if constexpr (MT <= 2) return launch_one<EPI, MT, 4>(nw, a, st, ev); break;
    case 7: if constexpr (MT == 1 && EPI == EPI_SWIGLU) return launch_one<EPI, MT, 7>(nw, a, st, ev); break;
    case 8: if constexpr (MT == 1 && (EPI == EPI_LOGITS || EPI == EPI_SWIGLU)) return launch_one<EPI, MT, 8>(nw, a, st, ev); break;
    case 9: if constexpr (MT == 1 && EPI == EPI_SWIGLU) return launch_one<EPI, MT, 9>(nw, a, st, ev); break;
    case 10: if constexpr (MT == 1 && EPI == EPI_SWIGLU) return launch_one<EPI, MT, 10>(nw, a, st, ev); break;
  }
  return hipErrorInvalidValue;
}

template <int EPI>
hipError_t launch_mt(int mt, int S, int nw, const GemmArgs& a, hipStream_t st, LaunchEvents ev) {
  switch (mt) {
    case 1: return launch_s<EPI, 1>(S, nw, a, st, ev);
    case 2: return launch_s<EPI, 2>(S, nw, a, st, ev);
    case 3: return launch_s<EPI, 3>(S, nw, a, st, ev);
    case 4: return launch_s<EPI, 4>(S, nw, a, st, ev);
  }
  return hipErrorInvalidValue;
}

// What launch_qkv_attn_any does for a shape: launch it, or report its
// co-resident workgroups (at `pre` preloaded gate/up iterations) or the
// largest `pre` its LDS holds.
struct FuseQuery {
  enum { LAUNCH, CAPACITY, PRE_MAX } what = LAUNCH;
  int pre = 0;
  int result = 0;
};

template <int MT, int S, int OKI, int SG>
constexpr size_t fuse_red_bytes() {   // (a fused down tile's [4][256] fits below the O units'; the gate/up
                                       // tile reduces in the preload area)
  return std::max((size_t)4 * S * MT * 256, OKI > 0 ? (size_t)8 * 2 * 256 : (size_t)0) * sizeof(float);
}

template <int MT, int S, int HD, int OKI, int SG, int SD>
hipError_t launch_qkv_attn_one(const GemmArgs& g, const AttnArgs& a, const FuseCtl& f, const GemmArgs& o,
                               const GemmArgs& gu, const GemmArgs& dn, hipStream_t st, LaunchEvents ev,
                               FuseQuery& q) {
  constexpr size_t red = fuse_red_bytes<MT, S, OKI, SG>();
  constexpr size_t iter = (size_t)4 * SG * 1024;            // one preloaded iteration
  // preloaded iterations that the attention arrays' static LDS holds (the
  // last ones of each workgroup; the attention workgroups load them there
  // after their attention)
  constexpr int stat_fit = SG > 0 ? (int)(sizeof(FusedStatLds<HD, SG>) / std::max<size_t>(iter, 1)) : 0;
  auto kern = k_qkv_attn<MT, S, HD, OKI, SG, SD>;
  const int pre = q.what == FuseQuery::LAUNCH ? std::max(f.gu_pre, f.gu_pre_q) : q.pre;
  // (at least one iteration's room: the gate/up tile's reduction)
  const size_t lds = red + (SG > 0 ? (size_t)std::max(pre - std::min(pre, stat_fit), 1) * iter : 0);
  if (q.what != FuseQuery::LAUNCH) {
    int dev = 0;
    hipDeviceProp_t prop;
    hipFuncAttributes attr;
    if (hipGetDevice(&dev) != hipSuccess || hipGetDeviceProperties(&prop, dev) != hipSuccess ||
        hipFuncGetAttributes(&attr, reinterpret_cast<const void*>(kern)) != hipSuccess)
      return hipErrorInvalidValue;
    const size_t room = (size_t)prop.maxSharedMemoryPerMultiProcessor;
    if (q.what == FuseQuery::PRE_MAX) {
      const size_t used = attr.sharedSizeBytes + red;
      q.result = SG > 0 && room > used ? (int)std::min<size_t>(kGuPreMax, (room - used) / iter + stat_fit) : 0;
      return hipSuccess;
    }
    if (attr.sharedSizeBytes + lds > room) return hipErrorInvalidValue;
    int per_cu = 0;
    if (hipFuncSetAttribute(reinterpret_cast<const void*>(kern), hipFuncAttributeMaxDynamicSharedMemorySize,
                            (int)(room - attr.sharedSizeBytes)) != hipSuccess ||
        hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kern, 512, lds) != hipSuccess)
      return hipErrorInvalidValue;
    q.result = per_cu * prop.multiProcessorCount;
    return hipSuccess;
  }
  FuseCtl fl = f;
  fl.gu_lds = (int)red;
  fl.gu_stat = stat_fit;
  const int grid = g.n_tiles + f.n_cons + f.o_extra;
  if (ev.start) {
    hipExtLaunchKernelGGL(kern, dim3(grid), dim3(512), (uint32_t)lds, st, ev.start, ev.stop, 0u, g, a, fl, o, gu, dn);
  } else {
    kern<<<grid, 512, lds, st>>>(g, a, fl, o, gu, dn);
  }
  return hipGetLastError();
}

template <int MT, int S, int HD>
hipError_t launch_qkv_attn_oki(int oki, int sg, int sd, const GemmArgs& g, const AttnArgs& a, const FuseCtl& f,
                               const GemmArgs& o, const GemmArgs& gu, const GemmArgs& dn, hipStream_t st,
                               LaunchEvents ev, FuseQuery& q) {
  if (oki == 0 && sg == 0 && sd == 0) return launch_qkv_attn_one<MT, S, HD, 0, 0, 0>(g, a, f, o, gu, dn, st, ev, q);
  if constexpr (MT == 1) {
    switch (oki * 1000 + sg * 10 + sd) {
      case 8000: return launch_qkv_attn_one<MT, S, HD, 8, 0, 0>(g, a, f, o, gu, dn, st, ev, q);
      case 8040: return launch_qkv_attn_one<MT, S, HD, 8, 4, 0>(g, a, f, o, gu, dn, st, ev, q);
      case 8070: return launch_qkv_attn_one<MT, S, HD, 8, 7, 0>(g, a, f, o, gu, dn, st, ev, q);
      case 8041: return launch_qkv_attn_one<MT, S, HD, 8, 4, 1>(g, a, f, o, gu, dn, st, ev, q);
      case 8071: return launch_qkv_attn_one<MT, S, HD, 8, 7, 1>(g, a, f, o, gu, dn, st, ev, q);
      case 16000: return launch_qkv_attn_one<MT, S, HD, 16, 0, 0>(g, a, f, o, gu, dn, st, ev, q);
      case 16040: return launch_qkv_attn_one<MT, S, HD, 16, 4, 0>(g, a, f, o, gu, dn, st, ev, q);
      case 16070: return launch_qkv_attn_one<MT, S, HD, 16, 7, 0>(g, a, f, o, gu, dn, st, ev, q);
      case 16041: return launch_qkv_attn_one<MT, S, HD, 16, 4, 1>(g, a, f, o, gu, dn, st, ev, q);
      case 16071: return launch_qkv_attn_one<MT, S, HD, 16, 7, 1>(g, a, f, o, gu, dn, st, ev, q);
    }
  }
  return hipErrorInvalidValue;
}

template <int MT, int S>
hipError_t launch_qkv_attn_hd(int hd, int oki, int sg, int sd, const GemmArgs& g, const AttnArgs& a,
                              const FuseCtl& f, const GemmArgs& o, const GemmArgs& gu, const GemmArgs& dn,
                              hipStream_t st, LaunchEvents ev, FuseQuery& q) {
  if (hd == 64) return launch_qkv_attn_oki<MT, S, 64>(oki, sg, sd, g, a, f, o, gu, dn, st, ev, q);
  if (hd == 128) return launch_qkv_attn_oki<MT, S, 128>(oki, sg, sd, g, a, f, o, gu, dn, st, ev, q);
  return hipErrorInvalidValue;
}

hipError_t launch_qkv_attn_any(int mt, int S, int hd, int oki, int sg, int sd, const GemmArgs& g, const AttnArgs& a,
                               const FuseCtl& f, const GemmArgs& o, const GemmArgs& gu, const GemmArgs& dn,
                               hipStream_t st, LaunchEvents ev, FuseQuery& q) {
  switch (mt * 4 + S) {
    case 1 * 4 + 1: return launch_qkv_attn_hd<1, 1>(hd, oki, sg, sd, g, a, f, o, gu, dn, st, ev, q);
    case 1 * 4 + 2: return launch_qkv_attn_hd<1, 2>(hd, oki, sg, sd, g, a, f, o, gu, dn, st, ev, q);
    case 2 * 4 + 1: return launch_qkv_attn_hd<2, 1>(hd, oki, sg, sd, g, a, f, o, gu, dn, st, ev, q);
    case 2 * 4 + 2: return launch_qkv_attn_hd<2, 2>(hd, oki, sg, sd, g, a, f, o, gu, dn, st, ev, q);
    case 3 * 4 + 1: return launch_qkv_attn_hd<3, 1>(hd, oki, sg, sd, g, a, f, o, gu, dn, st, ev, q);
    case 3 * 4 + 2: return launch_qkv_attn_hd<3, 2>(hd, oki, sg, sd, g, a, f, o, gu, dn, st, ev, q);
    case 4 * 4 + 1: return launch_qkv_attn_hd<4, 1>(hd, oki, sg, sd, g, a, f, o, gu, dn, st, ev, q);
    case 4 * 4 + 2: return launch_qkv_attn_hd<4, 2>(hd, oki, sg, sd, g, a, f, o, gu, dn, st, ev, q);
  }
  return hipErrorInvalidValue;
}

// k-blocks per wavefront of the fused O units for an O weight of kb k-blocks
// (0: no fused O; -1: unsupported)
int o_ki(int kb) { return kb == 0 ? 0 : kb <= 64 ? 8 : kb <= kFuseOMaxKb ? 16 : -1; }

}  // namespace

// Shape key of the fused launch queries (cached: the answers do not change,
// and nothing is asked during a graph capture once the engine has warmed up).
static int64_t fuse_key(int kind, int mt, int S, int head_dim, int oki, int sg, int sd, int pre) {
  return (((((((int64_t)kind * 8 + mt) * 4 + S) * 256 + head_dim) * 32 + oki) * 16 + sg) * 4 + sd) * 16 + pre;
}

static int fuse_query(int kind, int mt, int S, int head_dim, int oki, int sg, int sd, int pre) {
  static std::map<int64_t, int> cache;   // 0 or more: the answer; -1: unsupported
  const int64_t key = fuse_key(kind, mt, S, head_dim, oki, sg, sd, pre);
  auto it = cache.find(key);
  if (it != cache.end()) return it->second;
  FuseQuery q;
  q.what = kind == 0 ? FuseQuery::CAPACITY : FuseQuery::PRE_MAX;
  q.pre = pre;
  int r = -1;
  if (launch_qkv_attn_any(mt, S, head_dim, oki, sg, sd, GemmArgs{}, AttnArgs{}, FuseCtl{}, GemmArgs{}, GemmArgs{},
                          GemmArgs{}, nullptr, LaunchEvents{}, q) == hipSuccess)
    r = q.result;
  cache[key] = r;
  return r;
}

int qkv_attn_capacity(int mt, int S, int head_dim, int o_kb, int gu_S, int gu_pre, int d_S) {
  const int oki = o_ki(o_kb);
  if (mt < 1 || mt > 4 || S < 1 || S > 2 || (head_dim != 64 && head_dim != 128) || oki < 0 || (oki > 0 && mt != 1) ||
      (gu_S != 0 && gu_S != 4 && gu_S != 7) || (gu_S > 0 && (oki == 0 || gu_pre < 1 || gu_pre > kGuPreMax)) ||
      (d_S != 0 && (d_S != 1 || gu_S == 0)))
    return 0;
  const int r = fuse_query(0, mt, S, head_dim, oki, gu_S, d_S, gu_S > 0 ? gu_pre : 0);
  return r > 0 ? r : 0;
}

int qkv_attn_gu_pre_max(int S, int head_dim, int o_kb, int gu_S, int d_S) {
  const int oki = o_ki(o_kb);
  if (S < 1 || S > 2 || (head_dim != 64 && head_dim != 128) || oki <= 0 || (gu_S != 4 && gu_S != 7) ||
      (d_S != 0 && d_S != 1))
    return 0;
  const int r = fuse_query(1, 1, S, head_dim, oki, gu_S, d_S, 0);
  return r > 0 ? r : 0;
}

hipError_t launch_qkv_attn(int mt, int S, int head_dim, const GemmArgs& g, const AttnArgs& a, const FuseCtl& f,
                           const GemmArgs* o, const GemmArgs* gu, int gu_S, const GemmArgs* dn, hipStream_t st,
                           LaunchEvents ev) {
  // the GEMM tiles cover the strips exactly, one input range; the attention
  // part is the single-chunk plan with one query tile per workgroup
  if (g.n_tiles < 1 || g.ksplit != 1 || g.kb_split < g.kb_total || (size_t)g.n_tiles * S != (size_t)g.n_strips)
    return hipErrorInvalidValue;
  if (!a.wide || a.n_splits != 1 || a.nqt != 1 || a.split_len % 128 || a.n_seq < 1 || a.n_seq > kMaxPassSeqs)
    return hipErrorInvalidValue;
  if (!f.counters || !f.err || f.n_prod != g.n_tiles || f.n_cons != a.n_kv * a.n_qblocks * a.n_seq)
    return hipErrorInvalidValue;
  int oki = 0;
  const int workers = f.o_extra + f.n_prod;
  if (o) {
    // one row tile; O units: one strip each over one input range, every
    // worker with two units an extra workgroup
    oki = o_ki(o->kb_total);
    if (mt != 1 || oki <= 0 || o->n_strips != f.o_units || f.o_units < 1 || f.o_extra < 0 || f.o_two < 0 ||
        f.o_two > f.o_extra || f.o_units > workers + f.o_two || o->act_rows != a.act_rows || !o->A || !o->x ||
        !o->xg || !o->g_next || !o->ss_out || o->desc != a.desc)
      return hipErrorInvalidValue;
  } else if (f.o_units != 0 || f.o_extra != 0) {
    return hipErrorInvalidValue;
  }
  const int grid = g.n_tiles + f.n_cons + f.o_extra;
  if (gu) {
    // gate/up: needs the O units; tiles of gu_S strips cover the weight
    // exactly, one per workgroup of the grid at most; four wavefronts;
    // preloaded iterations within every wavefront's range
    if (!o || (gu_S != 4 && gu_S != 7) || gu->n_tiles != f.gu_tiles || f.gu_tiles < 1 || f.gu_tiles > grid ||
        (size_t)gu->n_tiles * gu_S != (size_t)gu->n_strips || gu->ksplit != 1 || gu->kb_split < gu->kb_total ||
        f.gu_pre < 1 || f.gu_pre_q < 0 || f.gu_pre > kGuPreMax || f.gu_pre_q > f.gu_pre || f.gu_pre > gu->kb_total / 4 ||
        f.n_odone != std::min(workers, f.o_units - f.o_two) || gu->act_rows != a.act_rows || gu->desc != a.desc ||
        gu->A != o->xg || gu->ss_in != o->ss_out)
      return hipErrorInvalidValue;
  } else if (f.gu_tiles != 0) {
    return hipErrorInvalidValue;
  }
  if (dn) {
    // down: needs gate/up; one strip per tile, one or two input ranges (each
    // unit, a tile's range, one workgroup of the grid at most); its input is
    // gate/up's output, its residual and outputs the O workers'
    if (!gu || dn->n_tiles * dn->ksplit != f.d_tiles || f.d_tiles < 1 || f.d_tiles > grid ||
        dn->n_tiles != dn->n_strips || dn->ksplit < 1 || dn->ksplit > 2 || dn->kb_split < 1 ||
        (dn->ksplit - 1) * dn->kb_split >= dn->kb_total || dn->ksplit * dn->kb_split < dn->kb_total ||
        dn->A != gu->out || dn->x != o->x || dn->xg != o->xg || dn->ss_out != o->ss_out || !dn->g_next ||
        dn->act_rows != a.act_rows || dn->desc != a.desc)
      return hipErrorInvalidValue;
    if (dn->ksplit > 1 && (!dn->part || !dn->counters || dn->n_tiles > kSplitCounters ||
                           (size_t)dn->n_tiles * dn->ksplit * 256 > kSplitPartFloats))
      return hipErrorInvalidValue;
  } else if (f.d_tiles != 0) {
    return hipErrorInvalidValue;
  }
  const int cap = qkv_attn_capacity(mt, S, head_dim, o ? o->kb_total : 0, gu ? gu_S : 0, gu ? f.gu_pre : 0,
                                    dn ? 1 : 0);
  if (cap <= 0 || grid > cap) return hipErrorInvalidValue;
  FuseQuery q;
  return launch_qkv_attn_any(mt, S, head_dim, oki, gu ? gu_S : 0, dn ? 1 : 0, g, a, f, o ? *o : GemmArgs{},
                             gu ? *gu : GemmArgs{}, dn ? *dn : GemmArgs{}, st, ev, q);
}

hipError_t launch_gemm(int epi, int mt, int S, int nw, const GemmArgs& a, hipStream_t st, LaunchEvents ev) {
  if (nw < 4 || nw > 8 || S < 1 || (size_t)nw * S * mt * 1024 > 64 * 1024) return hipErrorInvalidValue;
  // the tiles cover the strips; only gate/up workgroups of 8+ strips may be ragged
  if (a.n_tiles < 1 || (size_t)a.n_tiles * S < (size_t)a.n_strips || (size_t)(a.n_tiles - 1) * S >= (size_t)a.n_strips)
    return hipErrorInvalidValue;
  if (a.n_tiles * S != a.n_strips && !(epi == EPI_SWIGLU && mt == 1 && S >= 8)) return hipErrorInvalidValue;
  // split input: every range non-empty, partial tiles and counters supplied
  if (a.ksplit < 1 || a.kb_split < 1 || (a.ksplit - 1) * a.kb_split >= a.kb_total ||
      a.ksplit * a.kb_split < a.kb_total)
    return hipErrorInvalidValue;
  if (a.ksplit > 1 && (!a.part || !a.counters || a.n_tiles > kSplitCounters ||
                       (size_t)a.n_tiles * a.ksplit * S * mt * 256 > kSplitPartFloats))
    return hipErrorInvalidValue;
  switch (epi) {
    case EPI_QKV: return launch_mt<EPI_QKV>(mt, S, nw, a, st, ev);
    case EPI_RESID: return launch_mt<EPI_RESID>(mt, S, nw, a, st, ev);
    case EPI_SWIGLU: return launch_mt<EPI_SWIGLU>(mt, S, nw, a, st, ev);
    case EPI_LOGITS: return launch_mt<EPI_LOGITS>(mt, S, nw, a, st, ev);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_gemm_rows(int epi, const GemmArgs& a, hipStream_t st, LaunchEvents ev) {
  if (a.n_tiles < 1 || a.m_blocks < 1 || a.ksplit < 1 || a.ksplit > a.kb_total) return hipErrorInvalidValue;
  if (a.n_tiles * kRowsTileStrips < a.n_strips || (a.ksplit > 1 && !a.part)) return hipErrorInvalidValue;
  if ((size_t)a.n_tiles * a.m_blocks * a.ksplit >= (1u << 31)) return hipErrorInvalidValue;
  if (a.m_blocks * kRowTiles * 16 > kMaxPassRows + kRowTiles * 16) return hipErrorInvalidValue;
  switch (epi) {
    case EPI_QKV: return launch_rows<EPI_QKV>(a, st, ev);
    case EPI_RESID: return launch_rows<EPI_RESID>(a, st, ev);
    case EPI_SWIGLU: return launch_rows<EPI_SWIGLU>(a, st, ev);
    case EPI_LOGITS: return launch_rows<EPI_LOGITS>(a, st, ev);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_tail(const TailArgs& a, int n_seq, hipStream_t st) {
  if (n_seq < 1 || n_seq > kMaxPassSeqs) return hipErrorInvalidValue;
  k_lm_tail<<<n_seq, 1024, 0, st>>>(a);
  return hipGetLastError();
}

hipError_t launch_stage(const TailArgs& a, hipStream_t st) {
  k_stage<<<1, 256, 0, st>>>(a);
  return hipGetLastError();
}

}  // namespace pard
