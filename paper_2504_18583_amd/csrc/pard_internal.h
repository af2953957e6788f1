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
//     sits at act_index(row, k, slots), i.e. the row slots of one 32-column
//     block are contiguous (64 bytes per row), so the MFMA A fragment of one
//     k-block is one contiguous run of rows * 64 bytes.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace pard {

constexpr int kMaxK = 32;
constexpr int kMaxSampleVocab = 1 << 18;   // largest vocabulary speculative sampling supports
constexpr int kMaxRows = 64;          // rows of a pass served by the skinny GEMM (prefill chunk)
constexpr int kMaxPassRows = 512;     // rows of one forward pass over all of its sequences
constexpr int kMaxPassSeqs = 64;      // sequences in one pass
constexpr int kMaxLmRows = kMaxPassRows;
// row-block GEMM: a workgroup of kRowsWaves wavefronts computes kRowTiles*16
// rows x kRowsWaves*kRowsWaveStrips strips of 16 columns
constexpr int kRowTiles = 9;
constexpr int kRowsWaves = 4;
constexpr int kRowsWaveStrips = 4;
constexpr int kRowsTileStrips = kRowsWaves * kRowsWaveStrips;
constexpr int kRowsPartFloats = kRowsWaves * kRowTiles * kRowsWaveStrips * 256;   // one partial tile
constexpr int kBlock = 256;
// skinny GEMM with a split input dimension: tile counters and fp32 partial tiles
constexpr int kSplitCounters = 4096;
constexpr size_t kSplitPartFloats = (size_t)4 << 20;
constexpr int kAttnWaves = 4;      // wavefronts per attention workgroup
constexpr int kAttnChunk = 256;    // keys per attention workgroup (decode passes): two tiles per wavefront
constexpr int kAttnWideMaxKeys = 2048;   // decode passes up to this context: one 8-wave workgroup covers all keys
constexpr int kAttnBatchChunk = 1024;    // keys per chunk, row-block passes over several sequences
constexpr int kAttnLongChunkMax = 2048;   // longest key chunk of a decode pass over a long context
constexpr int kAttnDecodeWGs = 256;       // decode passes: chunks grow while the grid exceeds this
constexpr int kAttnWideQTiles64 = 1;     // query tiles per such workgroup at head_dim 64 (measured: 1 ahead of 2 and 4)
constexpr int kAttnRecords = 512;  // max (query group, key chunk) partial records per KV head and sequence

// Position of activation element (row, k) in a k-blocked buffer with `slots`
// row slots per 32-column block: kMaxRows for passes served by the skinny
// GEMM (so a decode pass's few rows stay close together), kMaxPassRows for the
// row-block GEMM's passes.
__host__ __device__ inline size_t act_index(int row, int k, int slots) {
  return ((size_t)(k >> 5) * slots + row) * 32 + (k & 31);
}

// Position of element (key, dim) in one KV head's K cache region.
__host__ __device__ inline size_t k_index(int key, int dim, int hd) {
  return (((size_t)(key >> 4) * (hd >> 5) + (dim >> 5)) * 64 + (key & 15) + 16 * ((dim & 31) >> 3)) * 8 +
         (dim & 7);
}

// Slot of key (pos % 32) inside its 32-key block of the transposed V cache:
// attention's P^T fragment holds keys {4g..4g+3, 16+4g..16+4g+3} in lane
// group g, so those eight keys are stored contiguously at 8g..8g+7.
__host__ __device__ inline int v_slot(int k) {
  return (k & 16) ? ((k & 12) << 1) + 4 + (k & 3) : ((k & 12) << 1) + (k & 3);
}

// SplitMix64 (Steele, Lea, Flood 2014): the state advances by kGamma before
// each output; mix64 is the output function.
constexpr uint64_t kGamma = 0x9E3779B97F4A7C15ull;
__host__ __device__ inline uint64_t mix64(uint64_t z) {
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}

// Random numbers of speculative sampling: the uniform in [0, 1) (24 bits) of
// (sequence slot, verify step `draw`, position j, purpose) -- output
// 4j + purpose of the stream seeded with output `draw` of the stream seeded
// with output `slot` of the stream seeded with `seed`.
enum Purpose { PURPOSE_DRAFT = 0, PURPOSE_KEEP = 1, PURPOSE_LAST = 2, PURPOSE_FIRST = 3 };
__host__ __device__ inline float sample_uniform(uint64_t seed, int slot, int draw, int j, int purpose) {
  uint64_t z = mix64(seed + ((uint64_t)slot + 1) * kGamma);
  z = mix64(z + ((uint64_t)draw + 1) * kGamma);
  z = mix64(z + ((uint64_t)(4 * j + purpose) + 1) * kGamma);
  return (float)(z >> 40) * (1.0f / 16777216.0f);
}

// fp16 bits of v, nearest even.
__device__ inline uint16_t f16_bits(float v) { return __builtin_bit_cast(uint16_t, (_Float16)v); }
// fp16 bits of an activation that feeds a GEMM or the KV cache.  A value that
// fp16 cannot hold (|v| >= 65520 rounds to infinity) or a NaN sets `bad`; the
// caller then sets the pass's range flag (flag_range), and the host reports
// the pass's results as invalid.
__device__ inline uint16_t f16_flagged(float v, bool& bad) {
  bad |= !(fabsf(v) < 65520.0f);
  return f16_bits(v);
}
__device__ inline void flag_range(bool bad, int* ovf) {
  if (bad && ovf) *ovf = 1;
}

// One sequence's share of a forward pass: rows [row0, row0 + n_rows) at
// positions pos0.., of which the first n_real carry real tokens (committed
// afterwards; the rest are the draft's mask rows); lm rows [lm0, lm0 +
// lm_rows) of the pass's compacted lm_head rows belong to it.
struct PassSeq {
  int slot;       // sequence slot (KV cache, decode state)
  int row0, n_rows, n_real, pos0;
  int lm0, lm_rows;
  int pad;
};

// Rows of the next forward pass of one model: one or several sequences, each
// a contiguous run of rows.  Written by the host (granular calls, prefill) or
// by the step tail of the previous pass (fused loop).
struct FwdDesc {
  int n_rows;                  // rows in the pass
  int n_seq;                   // sequences in the pass
  int n_lm;                    // rows fed to the lm_head
  int pad;
  PassSeq seq[kMaxPassSeqs];
  int ids[kMaxPassRows];       // token id of each row
  int pos[kMaxPassRows];       // absolute position of each row
  int slot[kMaxPassRows];      // sequence slot of each row
  int lm_src[kMaxPassRows];    // pass row of each lm row
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
  int vsd;                   // vanilla speculative decoding: K one-row draft passes per step
  int j;                     // draft passes done in the current step (vanilla)
  int draw;                  // verify steps since the prefill (speculative sampling's counter)
  float qM[kMaxK], qS[kMaxK];   // sampling: max logit and softmax normaliser of the draft's rows
};

// Device clock readings of the fused loop's pass boundaries (wall_clock64,
// constant rate): the first kernel of a pass stores its start, the step tails
// accumulate the draft, verify and accept phases and record each step's end.
constexpr int kStepRing = 4096;
struct PhaseClock {
  unsigned long long pass_start[2];   // [model]: start of its current pass
  unsigned long long tail_start;      // start of the current verify tail
  unsigned long long draft_ticks, verify_ticks, accept_ticks;
  unsigned long long n_steps;         // verify tails ended since the reset
  unsigned long long step_end[kStepRing];
};

enum Epi { EPI_QKV = 0, EPI_RESID = 1, EPI_SWIGLU = 2, EPI_LOGITS = 3 };
enum Tail { TAIL_NONE = 0, TAIL_PREFILL = 1, TAIL_DRAFT = 2, TAIL_VERIFY = 3, TAIL_VSD_DRAFT = 4 };

struct GemmArgs {
  const uint16_t* W;      // strip-packed weight (fp16 encoding)
  int kb_total;           // padded input dim / 32
  int n_tiles;            // output column tiles
  const uint16_t* A;      // fp16 activations, k-blocked (act_index), lda columns
  int lda;
  int act_rows;           // row slots of the pass's activation layout
  const FwdDesc* desc;   // rows: the pass's rows; EPI_LOGITS: its lm rows (row j reads pass row lm_src[j])
  // RMSNorm of the A operand (QKV, SWIGLU, LOGITS): A already holds x*g in
  // fp16; 1/rms comes from the producer's per-tile sums of squares.
  const float* ss_in; int ss_tiles;
  int ss_stride;          // floats between two rows' tile sums ([row][tile] layout, in and out)
  float eps, inv_k;
  // EPI_RESID: x += Y, and for the next consumer xg = fp16(x * g_next) and
  // per-tile sums of squares of x ([row][tile], ss_stride per row).
  float* x; int ldx;
  const float* g_next; uint16_t* xg; float* ss_out;
  // EPI_QKV / EPI_SWIGLU
  uint16_t* out; int ld_out;
  uint16_t* kc; uint16_t* vc; int cap;        // this layer's cache of slot 0
  size_t kv_seq_stride;                       // elements between two slots' caches
  const float* bias; const float2* rope;
  int q_dim, kv_dim, hd;
  // EPI_LOGITS: fp32 logits and the per-tile (max, argmax) of every lm row;
  // with samp_k = log2(e) / T > 0 also the per-tile sum of 2^((z - max) samp_k)
  float* logits; int vocab;
  float* amax_val; int* amax_idx; int amax_stride;   // entries per lm row
  float samp_k; float* amax_sum;
  // row-block GEMM (passes of more than kMaxRows rows): weight strips, row
  // blocks, input splits and the fp32 partial tiles of split inputs.  The
  // skinny GEMM splits its input into ksplit ranges of kb_split k-blocks
  // (ksplit = 1: one range) and counts arrivals per tile in counters (zero
  // between launches).
  int n_strips;
  int m_blocks, ksplit;
  float* part;
  int kb_split;
  int* counters;
  int* ovf;               // fp16 range flag of the activations this GEMM writes (f16_flagged), or null
};

// Second argmax pass over the lm_head tiles and the step tail: one workgroup
// per sequence of the pass.
struct TailArgs {
  const FwdDesc* desc;
  const float* amax_val; const int* amax_idx;
  int n_tiles, vocab;     // n_tiles: (max, argmax) entries per lm row
  int* result;            // argmax per lm row
  int tail;
  SeqState* states;       // decode state, indexed by slot
  int2* lm_map;           // per slot: (first lm row, lm rows) of the last pass
  int2* lm_map_draft;     // the draft's map (entries of sequences that leave a batch are cleared)
  FwdDesc* next_desc;     // staged by the tail (single-sequence passes) or k_stage
  int* out_tokens;        // emitted tokens of the fused loop, out_cap per slot (verify tail)
  int out_cap;
  // speculative sampling (samp_k = log2(e) / T > 0; 0: greedy): per-tile sums,
  // this model's logits (tile_w columns per tile), the draft's logits (verify)
  float samp_k;
  uint64_t seed;
  const float* amax_sum;
  const float* logits;
  const float* q_logits;
  int tile_w;
  PhaseClock* clock;      // pass-boundary clock (phase times of the fused loop)
};

struct AttnArgs {
  const uint16_t* q; int ldq;                 // [rows][H_q*hd] fp16, pair-interleaved dims
  const uint16_t* kc; const uint16_t* vc;     // this layer's cache of slot 0
  size_t kv_seq_stride;                       // elements between two slots' caches
  int cap;                                    // KV capacity (multiple of 32)
  uint16_t* out;                              // fp16, k-blocked (act_index), H_q*hd columns
  int act_rows;                               // row slots of the pass's activation layout
  const FwdDesc* desc;
  int n_heads, n_kv;
  int nqt, n_qblocks;                         // 16*nqt query pairs per workgroup, query groups per sequence
  int split_len, n_splits;                    // keys per chunk (multiple of 128), chunks
  int n_seq;                                  // sequences the grid covers (>= the pass's)
  float scale;
  float* part;                                // chunk records when n_splits > 1
  int wide;                                   // 1: one chunk per workgroup of 8 waves (n_splits == 1)
};

// A launch that carries the dependent phases of one decode layer: the QKV
// GEMM, the decode attention that reads its output and, optionally, the
// O-projection that reads the attention's output.  QKV workgroup b counts
// itself in on counter b % kFuseLanes once its stores are complete; attention
// workgroups wait for n_prod such arrivals in all (summing the kFuseLanes
// counters) and, when O units follow, count themselves in on each of the
// counters kFuseLanes .. 2 kFuseLanes - 1 once their own output stores are
// complete; O-projection worker b waits for n_cons arrivals on counter
// kFuseLanes + b % kFuseLanes alone (a few dozen arrivals awaited by hundreds
// of pollers: one line per poll, the pollers spread over the counters).
// Each layer of a model has its own set of counters, zeroed by the pass's
// embedding launch (k_embed), so no workgroup has to reset them at the end of
// a launch.  err is set if a wait exceeds its bounded spin.
//
// O units (o_units > 0): strip j of the O weight over its whole input range.
// Workers are the o_extra workgroups placed after the attention ones (they do
// nothing else, so their weight requests start with the launch), then the
// QKV workgroups; worker w < o_two takes units 2w and 2w + 1, a later worker
// unit o_two + w (if any).
//
// Gate/up units (gu_tiles > 0, with O units): workgroup b < gu_tiles runs
// gate/up tile b.  Its first gu_pre (gu_pre_q for QKV workgroups, which load
// theirs only once their tile is done) input iterations of weights are loaded
// straight into LDS early, while the attention runs; O workers count
// themselves in on counter 2 kFuseLanes + w % kFuseLanes once their
// epilogue's device-scope stores are complete, and the gate/up tiles wait for
// n_odone such arrivals before reading the O-projection's output (at device
// scope).
//
// Down tiles (d_tiles > 0, with gate/up): workgroup b < d_tiles runs down
// tile b once every gate/up tile has counted itself in on counter
// 3 kFuseLanes + t % kFuseLanes (h stored at device scope).
constexpr int kFuseLanes = 8;      // arrival counters per phase (spread over XCDs and memory channels)
constexpr int kFuseStride = 64;    // ints between two counters
constexpr int kFuseInts = 4 * kFuseLanes * kFuseStride;   // one layer's set: QKV, attention, O, gate/up arrivals
struct FuseCtl {
  int* counters = nullptr;         // this layer's kFuseInts ints, zero at the launch
  int n_prod = 0, n_cons = 0;      // QKV workgroups, attention workgroups
  int* err = nullptr;
  int o_units = 0, o_extra = 0, o_two = 0;
  int gu_tiles = 0, gu_pre = 0, gu_pre_q = 0;
  int n_odone = 0;                 // O workers with units
  int d_tiles = 0;
  int gu_lds = 0;                  // byte offset of the preloaded weights in the dynamic LDS (set by the launcher)
  int gu_stat = 0;                 // the last preloaded iterations of a workgroup that go into the attention
                                   // arrays' LDS instead (at most this many; set by the launcher)
};

// Optional timing events of one launch (recorded at the kernel's start and end).
struct LaunchEvents {
  hipEvent_t start = nullptr, stop = nullptr;
};

// COD training-data processing (one workgroup per sample).
struct CodArgs {
  int k_max;
  double r, r_min;         // retention decay and floor (float64: they decide the kept counts)
  int mask_id;
  uint64_t seed;
  int32_t *ids, *labels, *pos, *section, *column;   // packed outputs
  int32_t* out_len;                                 // packed length per sample
};

// Launchers (return hipSuccess or the launch error).
hipError_t launch_gemm(int epi, int mt, int S, int nw, const GemmArgs& a, hipStream_t st,
                       LaunchEvents ev = LaunchEvents{});
hipError_t launch_gemm_rows(int epi, const GemmArgs& a, hipStream_t st, LaunchEvents ev = LaunchEvents{});
// QKV GEMM (mt row tiles, S strips per workgroup, one input range) and the
// single-chunk decode attention reading its output, in one launch; only when
// every workgroup of it is co-resident (qkv_attn_capacity: workgroups the
// device holds at once, 0 if the shape has no fused kernel).
// With o (non-null, one row tile only) the launch also carries the
// O-projection + residual of the attention output (EPI_RESID, one strip per
// tile, one input range of at most kFuseOMaxKb k-blocks; f's O fields set).
// With gu as well (o required; f's gate/up fields set) it carries the
// gate/up GEMM (EPI_SWIGLU, gu_S strips per tile, one input range, four
// wavefronts), its first weight blocks preloaded into LDS; with dn as well
// (gu required) the down projection + residual (EPI_RESID, one strip per
// tile, one input range, four wavefronts; d_S = 1 in the queries).
constexpr int kFuseOMaxKb = 128;
int qkv_attn_capacity(int mt, int S, int head_dim, int o_kb = 0, int gu_S = 0, int gu_pre = 0, int d_S = 0);
// largest gu_pre the LDS holds for this launch shape (0: none)
int qkv_attn_gu_pre_max(int S, int head_dim, int o_kb, int gu_S, int d_S = 0);
hipError_t launch_qkv_attn(int mt, int S, int head_dim, const GemmArgs& g, const AttnArgs& a, const FuseCtl& f,
                           const GemmArgs* o, const GemmArgs* gu, int gu_S, const GemmArgs* dn, hipStream_t st,
                           LaunchEvents ev = LaunchEvents{});
hipError_t launch_tail(const TailArgs& a, int n_seq, hipStream_t st);
hipError_t launch_stage(const TailArgs& a, hipStream_t st);
hipError_t launch_attention(int head_dim, const AttnArgs& a, hipStream_t st);
size_t attn_part_floats(int head_dim, int nqt);
int attn_max_q_tiles(int head_dim);
hipError_t launch_cod(const int32_t* tokens, const int64_t* tok_off, const int64_t* out_off, int n_samples,
                      int max_columns, const CodArgs& a, hipStream_t st);
int cod_max_columns();

}  // namespace pard
