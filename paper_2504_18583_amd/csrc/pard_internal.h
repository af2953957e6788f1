// Internal structures shared by the engine (host) and the HIP kernels.
//
// Device data layout (all carved from the caller's arena):
//   * every weight matrix W [out, in] holds the model's bf16 values in fp16
//     encoding (exact for |w| >= 2^-14, smaller ones round to fp16
//     subnormals within 2^-25), so the fp16 MFMAs read it directly.  It is
//     stored in 1 KiB blocks of 16
//     output rows ("strip") x 32 input columns ("k-block"), each laid out in
//     the lane order of the v_mfma_f32_16x16x32_bf16 B operand (lane l holds
//     row l%16, columns 8*(l/16) .. +7).  Blocks are k-block-major: block
//     (kb, strip) sits at (kb * n_strips + strip) KiB, so while every
//     workgroup streams its strips, the grid as a whole sweeps contiguous
//     memory (spreading the reads over all HBM channels).
//   * Q/K rows are stored pair-interleaved per head (packed row 2j = dim j,
//     2j+1 = dim j + head_dim/2) so the rotate-half rotary pairs sit in
//     neighbouring lanes; K is cached in that order and attention's q.k is
//     invariant to it.  Gate/up rows are interleaved by strips (gate strip,
//     up strip, ...) so one tile holds matching gate and up columns.
//   * KV cache, fp16, per [batch][layer][kv_head] a region of cap keys:
//     K in blocks of 16 keys, each stored as head_dim/32 MFMA A-operand
//     fragments of 1 KiB (k_index); V in blocks of 32 keys stored transposed
//     ([dim][key slot], see the attention kernel), so both are read as
//     contiguous 1 KiB wavefront loads.
//   * activations that feed a GEMM (x*g, attention output, silu(gate)*up) are
//     fp16 and the GEMMs run fp16 MFMAs: a 10-bit mantissa on the activation
//     side (bf16 activations drift past the logit tolerance at 8B width and
//     depth).  They are k-blocked: element (row, k)
//     sits at act_index(row, k), i.e. the 64 row slots of one 32-column block
//     are contiguous (64 bytes per row), so the MFMA A fragment of one k-block
//     is one contiguous run of rows * 64 bytes.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace pard {

constexpr int kMaxK = 32;
constexpr int kMaxRows = 64;      // rows of one forward pass (prefill chunk, 2*max_k)
constexpr int kMaxLmRows = kMaxK + 1;
constexpr int kBlock = 256;
constexpr int kAttnWaves = 4;      // wavefronts per attention workgroup
constexpr int kAttnChunk = 256;    // keys per attention workgroup (decode passes): two tiles per wavefront
constexpr int kAttnRecords = 512;  // max (query group, key chunk) partial records per KV head

// Position of activation element (row, k) in a k-blocked [kMaxRows x K] buffer.
__host__ __device__ inline size_t act_index(int row, int k) {
  return ((size_t)(k >> 5) * kMaxRows + row) * 32 + (k & 31);
}

// Position of element (key, dim) in one KV head's K cache region.
__host__ __device__ inline size_t k_index(int key, int dim, int hd) {
  return (((size_t)(key >> 4) * (hd >> 5) + (dim >> 5)) * 64 + (key & 15) + 16 * ((dim & 31) >> 3)) * 8 +
         (dim & 7);
}

// fp16 bits of v, nearest even.
__device__ inline uint16_t f16_bits(float v) { return __builtin_bit_cast(uint16_t, (_Float16)v); }

// Rows of the next forward pass of one model.  Written by the host (granular
// calls) or by the tail of the previous pass (fused loop).
struct FwdDesc {
  int n_rows;     // rows in the pass
  int n_real;     // leading rows that carry real tokens (committed afterwards)
  int pos0;       // absolute position of row 0 (= committed KV length)
  int lm_row0;    // first row fed to the lm_head
  int lm_rows;    // rows fed to the lm_head
  int pad[3];
  int ids[kMaxRows];
};

// Decode state of one sequence slot.
struct SeqState {
  int L[2];                  // committed KV length: [0] target, [1] draft
  int k;                     // draft length of the current step
  int n_pending;             // tokens produced but not yet in the draft cache
  int pending[kMaxK + 1];
  int cand[kMaxK];           // draft candidates of the current step
  int t[kMaxK + 1];          // target argmax of the last verify pass
  int a, bonus;              // accepted count, bonus (= pending token for the target)
  int n_out, n_target;       // tokens written to the output buffer / requested
  int steps;
  int mask_id;
  int accept_hist[kMaxK + 1];
};

enum Epi { EPI_QKV = 0, EPI_RESID = 1, EPI_SWIGLU = 2, EPI_LOGITS = 3 };
enum Tail { TAIL_NONE = 0, TAIL_PREFILL = 1, TAIL_DRAFT = 2, TAIL_VERIFY = 3 };

struct GemmArgs {
  const uint16_t* W;      // strip-packed bf16 weight
  int kb_total;           // padded input dim / 32
  int n_tiles;            // output tiles (S strips each) = grid size
  const uint16_t* A;      // fp16 activations, k-blocked (act_index), lda columns
  int lda;
  const FwdDesc* desc;
  int lm_mode;            // 0: rows [0, n_rows)   1: rows [lm_row0, lm_row0 + lm_rows)
  // RMSNorm of the A operand (QKV, SWIGLU, LOGITS): A already holds x*g in
  // bf16; 1/rms comes from the producer's per-tile sums of squares.
  const float* ss_in; int ss_tiles;
  float eps, inv_k;
  // EPI_RESID: x += Y, and for the next consumer xg = bf16(x * g_next) and
  // per-tile sums of squares of x.
  float* x; int ldx;
  const float* g_next; uint16_t* xg; float* ss_out;
  // EPI_QKV / EPI_SWIGLU
  uint16_t* out; int ld_out;
  uint16_t* kc; uint16_t* vc; int cap;
  const float* bias; const float2* rope;
  int q_dim, kv_dim, hd;
  // EPI_LOGITS: fp32 logits and the per-tile (max, argmax) of every lm row
  float* logits; int vocab;
  float* amax_val; int* amax_idx;
};

// Second argmax pass over the lm_head tiles and the step tail (one workgroup).
struct TailArgs {
  const FwdDesc* desc;
  const float* amax_val; const int* amax_idx;
  int n_tiles, vocab;
  int* result;            // argmax per lm row
  int tail;
  SeqState* seq;
  FwdDesc* next_desc;     // staged by the tail
  int* out_tokens;        // emitted tokens of the fused loop (verify tail)
  int out_cap;
};

struct AttnArgs {
  const uint16_t* q; int ldq;                 // [rows][H_q*hd] fp16, pair-interleaved dims
  const uint16_t* kc; const uint16_t* vc;     // this layer's cache of one sequence
  int cap;                                    // KV capacity (multiple of 32)
  uint16_t* out;                              // fp16, k-blocked (act_index), H_q*hd columns
  const FwdDesc* desc;
  int n_heads, n_kv;
  int nqt, n_qblocks;                         // 16*nqt query pairs per workgroup, query groups
  int split_len, n_splits;                    // keys per chunk (multiple of 128), chunks
  float scale;
  float* part;                                // chunk records when n_splits > 1
};

// Optional timing events of one launch (recorded at the kernel's start and end).
struct LaunchEvents {
  hipEvent_t start = nullptr, stop = nullptr;
};

// Launchers (return hipSuccess or the launch error).
hipError_t launch_gemm(int epi, int mt, int S, int nw, const GemmArgs& a, hipStream_t st,
                       LaunchEvents ev = LaunchEvents{});
hipError_t launch_tail(const TailArgs& a, hipStream_t st);
hipError_t launch_attention(int head_dim, const AttnArgs& a, hipStream_t st);
size_t attn_part_floats(int head_dim, int nqt);
int attn_max_q_tiles(int head_dim);

}  // namespace pard
