// Launchers of the load-time kernels and the embedding gather.
#pragma once

#include "pard_internal.h"

namespace pard {

enum RowMap { MAP_IDENTITY = 0, MAP_QKV = 1, MAP_GATEUP = 2 };

// Generation of one strip-packed weight (or a fused pair/triple of weights).
struct GenArgs {
  uint16_t* dst;
  int n_strips, kb_total;   // packed shape: n_strips*16 rows x kb_total*32 cols
  int rows, cols;           // canonical rows (per tensor) and columns
  int map;                  // RowMap
  int q_dim, kv_dim, hd;    // MAP_QKV
  uint64_t key0, key1, key2;
  double stdv;
};

hipError_t launch_gen_packed(const GenArgs& a, hipStream_t st);
hipError_t launch_gen_bias(const GenArgs& a, float* dst, int n_total, hipStream_t st);
hipError_t launch_fill_f32(float* p, size_t n, float v, hipStream_t st);
hipError_t launch_fill_u32(uint32_t* p, size_t n, uint32_t v, hipStream_t st);
// LLaMA-3.1-style rotary frequency scaling (factor 0: none).
struct RopeScaling {
  double factor = 0.0, low = 1.0, high = 1.0, orig = 1.0;
};
hipError_t launch_rope_table(float2* tab, int cap, int hd, double theta, const RopeScaling& sc, hipStream_t st);
// t_start (may be null): receives the device clock at the kernel's start (the
// start of the pass).  fuse_cnt (may be null): n_sets fused-launch counter
// sets (kFuseInts ints each) to zero.  ovf: fp16 range flag (f16_flagged).
hipError_t launch_embed(const uint16_t* E, int n_strips, int d, const FwdDesc* desc, float* x, const float* g,
                        uint16_t* xg, int act_rows, float* ss, int ss_stride, int max_rows,
                        unsigned long long* t_start, int* fuse_cnt, int n_sets, int* ovf, hipStream_t st);
hipError_t launch_gather_u16(const uint16_t* src, const size_t* idx, int n, float* out, hipStream_t st);

}  // namespace pard
