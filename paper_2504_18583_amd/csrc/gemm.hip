// Skinny bf16 GEMM for decode-sized row counts, on gfx950 MFMA.
//
//   Y[r, n] = sum_k A[r, k] * W[n, k]            (W block-packed, A fp16)
//
// Decode streams every weight once per forward (Sec. 2.1: decoding is bound by
// reloading the weights), so the kernel is organised around the weight
// stream.  A workgroup owns S strips (16 output columns each) over the whole
// input dimension; its NW wavefronts split the input dimension, each one
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
// Epilogues fuse the surrounding element-wise work of a Llama block:
//   EPI_QKV     RMSNorm row scale (A holds x*g in fp16, written by the
//               producer; 1/rms comes from the producer's per-tile sums of
//               squares), bias, rotate-half RoPE on Q/K, Q to an fp16 buffer,
//               K (16-key MFMA fragments) and V (32-key blocks, transposed)
//               to the fp16 cache.
//   EPI_RESID   x += Y (O-projection, down-projection), plus fp16(x * g_next)
//               and per-tile row sums of squares for the next normalised GEMM.
//   EPI_SWIGLU  RMSNorm row scale, h = silu(gate) * up, fp16.
//   EPI_LOGITS  final RMSNorm scale, fp32 logits and per-tile (max, argmax).
// k_lm_tail then reduces the tiles per row (lowest id on ties) and runs the
// step tail: candidates for a draft pass; greedy prefix acceptance, KV
// rollback and next-pass staging for a verify pass.
#include "pard_internal.h"

#include <hip/hip_ext.h>

#include <climits>

namespace pard {
namespace {

typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));



constexpr int kRsrcWord3 = 0x00020000;   // buffer descriptor word 3 for gfx9-family raw buffers
constexpr int kCachePolicyNT = 2;        // non-temporal: weights are streamed once

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

// Slot of key (pos % 32) inside its 32-key block of the transposed V cache:
// attention's P^T fragment holds keys {4g..4g+3, 16+4g..16+4g+3} in lane
// group g, so those eight keys are stored contiguously at 8g..8g+7.
__device__ __forceinline__ int v_slot(int k) {
  return (k & 16) ? ((k & 12) << 1) + 4 + (k & 3) : ((k & 12) << 1) + (k & 3);
}

template <int MT, int S, int EPI>
__global__ __launch_bounds__(512) void k_gemm(const GemmArgs p) {
  constexpr int NE = S * MT * 256;   // elements of one workgroup tile
  constexpr int NJ = S * MT;         // elements per thread in the epilogue (first 256 threads)
  // k-blocks per pipeline stage: 8 KiB of W per wave (smaller for prefill-sized row counts)
  constexpr int U = MT >= 3 ? 2 : ((8 / S) > 0 ? 8 / S : 1);
  extern __shared__ float red[];     // [NW][NE]
  __shared__ float rs_s[MT * 16];

  const int tile = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & 63;
  const int nw = blockDim.x >> 6;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // uniform per wavefront

  // wave w streams k-blocks w, w + nw, w + 2*nw, ...: at any time the
  // workgroup reads nw consecutive k-blocks of each strip
  const int n_it = (p.kb_total - wave + nw - 1) / nw;

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
  const int n_strips = p.n_tiles * S;
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
      const int kb = wave + min(its + u, n_it - 1) * nw;
#pragma unroll
      for (int s = 0; s < S; ++s)
        w[u][s] = __builtin_amdgcn_raw_buffer_load_b128(wrs, w_voff, (kb * n_strips + s) * 1024, kCachePolicyNT);
    }
  };

  // The weight stream does not depend on the pass: its first stage is in
  // flight before the pass descriptor is read.
  if (n_it > 0) load_w(w0, 0);
  __builtin_amdgcn_sched_barrier(0);

  const FwdDesc d = *p.desc;
  const int row_begin = p.lm_mode ? d.lm_row0 : 0;
  const int row_count = p.lm_mode ? d.lm_rows : d.n_rows;

  // A fragment of this lane: row (lane % 16) of each M tile, 8 columns at
  // 8*(lane/16); A is k-blocked, so k-block kb of all rows is one contiguous
  // run at kb * kMaxRows * 64 bytes.  Rows past the pass get an offset beyond
  // the buffer: the hardware returns zeros for them without a memory access.
  const __amdgpu_buffer_rsrc_t ars = __builtin_amdgcn_make_buffer_rsrc(
      const_cast<uint16_t*>(p.A), 0, kMaxRows * p.lda * 2, kRsrcWord3);
  constexpr int kOutOfRange = 0x7FFFFFF0;
  int a_voff[MT];
#pragma unroll
  for (int mt = 0; mt < MT; ++mt) {
    const int r = mt * 16 + (lane & 15);
    a_voff[mt] = r < row_count ? (row_begin + r) * 64 + (lane >> 4) * 16 : kOutOfRange;
  }
  auto load_a = [&](u32x4 (&a)[U][MT], int its) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int kb = wave + min(its + u, n_it - 1) * nw;
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
        a[u][mt] = __builtin_amdgcn_raw_buffer_load_b128(ars, a_voff[mt], kb * (kMaxRows * 64), 0);
    }
  };
  auto load = [&](u32x4 (&w)[U][S], u32x4 (&a)[U][MT], int its) {
    load_w(w, its);
    load_a(a, its);
  };

  // thread tid (< 256) of the epilogue owns, for j = s*MT + mt, element
  // (row, col) below; its epilogue operands are fetched while the weights stream
  const bool epi = tid < 256;
  const int ew = tid >> 6;
  const int rsub = (lane >> 4) * 4 + ew;
  const int csub = lane & 15;
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
          e0[j] = p.x[(size_t)(row_begin + row) * p.ldx + n];
          e1[j] = p.g_next[n];
        }
      } else if constexpr (EPI == EPI_QKV) {
        if (epi && p.bias) e0[j] = p.bias[n];
        if (epi && row < row_count && n < p.q_dim + p.kv_dim)
          e2[j] = p.rope[(size_t)(d.pos0 + row) * (p.hd / 2) + ((n % p.hd) >> 1)];
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

  // 1/rms per row from the producer's per-tile sums of squares: 16 threads per
  // row, 16 independent loads each in flight together, fixed summation order
  auto row_scales = [&]() {
    if (tid < 256) {
      for (int r = tid >> 4; r < MT * 16; r += 16) {
        const int row = min(row_begin + r, kMaxRows - 1);
        float t = 0.f;
        for (int q0 = tid & 15; q0 < p.ss_tiles; q0 += 256) {
          float part[16];
#pragma unroll
          for (int u = 0; u < 16; ++u) {
            const int q = q0 + 16 * u;
            part[u] = q < p.ss_tiles ? p.ss_in[(size_t)q * kMaxRows + row] : 0.f;
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
  if (n_it > 0) {
    int its = 0;
    load_a(a0, its);
    __builtin_amdgcn_sched_barrier(0);
    if constexpr (EPI != EPI_RESID) row_scales();   // overlaps the first weight loads
    load(w1, a1, its + U);
    __builtin_amdgcn_sched_barrier(0);
    prefetch_epilogue();
    __builtin_amdgcn_sched_barrier(0);
    while (true) {
      compute(w0, a0, its);
      __builtin_amdgcn_sched_barrier(0);
      its += U;
      if (its >= n_it) break;
      load(w0, a0, its + U);
      __builtin_amdgcn_sched_barrier(0);
      compute(w1, a1, its);
      __builtin_amdgcn_sched_barrier(0);
      its += U;
      if (its >= n_it) break;
      load(w1, a1, its + U);
      __builtin_amdgcn_sched_barrier(0);
    }
  } else {
    if constexpr (EPI != EPI_RESID) row_scales();
    prefetch_epilogue();
  }

  // ---- workgroup reduction over the NW input-dimension slices (wave order) ----
#pragma unroll
  for (int s = 0; s < S; ++s)
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int i = 0; i < 4; ++i) red[wave * NE + ((s * MT + mt) * 4 + i) * 64 + lane] = acc[s][mt][i];

  __syncthreads();

  // the first four wavefronts run the epilogue; all waves stay until the end
  // so that every barrier below is reached by the whole workgroup
  float v[NJ];
#pragma unroll
  for (int j = 0; j < NJ; ++j) {
    const int e = j * 256 + (tid & 255);
    float t = red[e];
    for (int w = 1; w < nw; ++w) t += red[w * NE + e];
    v[j] = t;
  }

  if constexpr (EPI == EPI_QKV) {
    if (!epi) return;   // no barrier follows in this epilogue
    const int pos0 = d.pos0;
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const int s = j / MT, mt = j % MT;
      const int row = mt * 16 + rsub;
      const int n = (tile * S + s) * 16 + csub;
      float y = v[j] * rs_s[row] + e0[j];            // + bias
      const float partner = __shfl_xor(y, 1);
      if (row < row_count) {
        const int pos = pos0 + row;
        if (n < p.q_dim + p.kv_dim) {
          const float2 cs = e2[j];                     // rotary (cos, sin) of (pos, pair)
          y = (n & 1) ? (y * cs.x + partner * cs.y) : (y * cs.x - partner * cs.y);
        }
        const uint16_t b = f16_bits(y);
        if (n < p.q_dim) {
          p.out[(size_t)row * p.ld_out + n] = b;
        } else if (n < p.q_dim + p.kv_dim) {
          const int c = n - p.q_dim;
          p.kc[(size_t)(c / p.hd) * p.cap * p.hd + k_index(pos, c % p.hd, p.hd)] = b;
        } else {
          const int c = n - p.q_dim - p.kv_dim;
          const size_t blk = (size_t)(c / p.hd) * (p.cap / 32) + (pos >> 5);
          p.vc[(blk * p.hd + (c % p.hd)) * 32 + v_slot(pos & 31)] = b;
        }
      }
    }
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
        const size_t o = (size_t)(row_begin + row) * p.ldx + n;
        const float xn = e0[j] + v[j];                 // residual + projection
        p.x[o] = xn;
        p.xg[act_index(row_begin + row, n)] = f16_bits(xn * e1[j]);
        sq[mt] += xn * xn;
      }
    }
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      const float t = sum16(sq[mt]);
      if (csub == 0) p.ss_out[(size_t)tile * kMaxRows + mt * 16 + rsub] = t;
    }
  } else if constexpr (EPI == EPI_SWIGLU) {
    if (!epi) return;   // no barrier follows in this epilogue
#pragma unroll
    for (int q = 0; q < S / 2; ++q)
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        const int row = mt * 16 + rsub;
        const float gt = v[(2 * q) * MT + mt] * rs_s[row];
        const float up = v[(2 * q + 1) * MT + mt] * rs_s[row];
        const float h = gt / (1.0f + expf(-gt)) * up;
        const int f = (tile * (S / 2) + q) * 16 + csub;
        if (row < row_count) p.out[act_index(row, f)] = f16_bits(h);
      }
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
        p.amax_val[(size_t)r * p.n_tiles + tile] = bv;
        p.amax_idx[(size_t)r * p.n_tiles + tile] = (bi == INT_MAX) ? INT_MAX : tile * TW + bi;
      }
    }
  }
}

// Step tail, run by one thread once every argmax of the pass is known.
__device__ void run_tail(const TailArgs& p, const FwdDesc& d, const int* res) {
  SeqState* s = p.seq;
  if (p.tail == TAIL_PREFILL) {
    s->bonus = res[0];
    s->t[0] = res[0];
    s->pending[0] = res[0];
    s->n_pending = 1;
  } else if (p.tail == TAIL_DRAFT) {
    const int k = s->k;
    for (int i = 0; i < k; ++i) s->cand[i] = res[i];
    s->L[1] = d.pos0 + d.n_real;                   // mask rows are not committed
    FwdDesc* nd = p.next_desc;                      // verify pass: [pending, c_1..c_k]
    nd->ids[0] = s->bonus;
    for (int i = 0; i < k; ++i) nd->ids[1 + i] = res[i];
    nd->n_rows = k + 1;
    nd->n_real = k + 1;
    nd->pos0 = s->L[0];
    nd->lm_row0 = 0;
    nd->lm_rows = k + 1;
  } else if (p.tail == TAIL_VERIFY) {
    const int k = s->k;
    int a = 0;
    while (a < k && s->cand[a] == res[a]) ++a;      // longest agreeing prefix
    const int bonus = res[a];
    for (int i = 0; i <= k; ++i) s->t[i] = res[i];
    s->a = a;
    s->bonus = bonus;
    s->L[0] = d.pos0 + a + 1;                      // keep pending + accepted rows
    for (int i = 0; i < a; ++i) s->pending[i] = s->cand[i];
    s->pending[a] = bonus;
    s->n_pending = a + 1;
    if (p.out_tokens) {
      for (int i = 0; i <= a; ++i) {
        if (s->n_out < p.out_cap) p.out_tokens[s->n_out] = s->pending[i];
        ++s->n_out;
      }
    }
    ++s->steps;
    ++s->accept_hist[a];
    FwdDesc* nd = p.next_desc;
    if (k > 0) {                                    // next draft: pending + k-1 masks
      int n = 0;
      for (int i = 0; i <= a; ++i) nd->ids[n++] = s->pending[i];
      for (int i = 0; i < k - 1; ++i) nd->ids[n++] = s->mask_id;
      nd->n_rows = n;
      nd->n_real = a + 1;
      nd->pos0 = s->L[1];
      nd->lm_row0 = a;
      nd->lm_rows = k;
    } else {                                        // plain target step
      nd->ids[0] = bonus;
      nd->n_rows = 1;
      nd->n_real = 1;
      nd->pos0 = s->L[0];
      nd->lm_row0 = 0;
      nd->lm_rows = 1;
    }
  }
}

// One workgroup of 1024 threads: wave w reduces lm rows w, w+16, ... over
// tiles, 16 independent loads per lane in flight at a time.
__global__ __launch_bounds__(1024) void k_lm_tail(const TailArgs p) {
  __shared__ int res_s[kMaxLmRows];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const FwdDesc d = *p.desc;
  const int rows = d.lm_rows;
  for (int r = wave; r < rows; r += 16) {
    float bv = -INFINITY;
    int bi = INT_MAX;
    const float* vals = p.amax_val + (size_t)r * p.n_tiles;
    const int* idxs = p.amax_idx + (size_t)r * p.n_tiles;
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
  __syncthreads();
  if (tid == 0) {
    for (int r = 0; r < rows; ++r) p.result[r] = res_s[r];
    run_tail(p, d, res_s);
  }
}

template <int EPI, int MT, int S>
hipError_t launch_one(int nw, const GemmArgs& a, hipStream_t st, LaunchEvents ev) {
  const size_t lds = (size_t)nw * S * MT * 256 * sizeof(float);
  if (nw > 8) return hipErrorInvalidValue;
  if (ev.start) {
    hipExtLaunchKernelGGL(k_gemm<MT, S, EPI>, dim3(a.n_tiles), dim3(64 * nw), (uint32_t)lds, st, ev.start, ev.stop,
                          0u, a);
  } else {
    k_gemm<MT, S, EPI><<<dim3(a.n_tiles), dim3(64 * nw), lds, st>>>(a);
  }
  return hipGetLastError();
}

template <int EPI, int MT>
hipError_t launch_s(int S, int nw, const GemmArgs& a, hipStream_t st, LaunchEvents ev) {
  switch (S) {
    case 1: if constexpr (EPI != EPI_SWIGLU) return launch_one<EPI, MT, 1>(nw, a, st, ev); break;
    case 2: return launch_one<EPI, MT, 2>(nw, a, st, ev);
    case 4: if constexpr (MT <= 2) return launch_one<EPI, MT, 4>(nw, a, st, ev); break;
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

}  // namespace

hipError_t launch_gemm(int epi, int mt, int S, int nw, const GemmArgs& a, hipStream_t st, LaunchEvents ev) {
  if (nw < 4 || nw > 8 || (size_t)nw * S * mt * 1024 > 32 * 1024) return hipErrorInvalidValue;
  switch (epi) {
    case EPI_QKV: return launch_mt<EPI_QKV>(mt, S, nw, a, st, ev);
    case EPI_RESID: return launch_mt<EPI_RESID>(mt, S, nw, a, st, ev);
    case EPI_SWIGLU: return launch_mt<EPI_SWIGLU>(mt, S, nw, a, st, ev);
    case EPI_LOGITS: return launch_mt<EPI_LOGITS>(mt, S, nw, a, st, ev);
  }
  return hipErrorInvalidValue;
}

hipError_t launch_tail(const TailArgs& a, hipStream_t st) {
  k_lm_tail<<<1, 1024, 0, st>>>(a);
  return hipGetLastError();
}

}  // namespace pard
