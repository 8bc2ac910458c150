// Internal interface between the C-ABI host code and the HIP kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace pda {

constexpr int kStep = 32;                 // tokens per pipeline step of a wave
constexpr int kMaxWaves = 8;              // waves per attention workgroup (at most)
constexpr int kMaxBlockThreads = 64 * kMaxWaves;
// Waves per attention workgroup at most for a head size: a wave of D = 256
// holds 32 KB of K/V per step in registers, twice the D = 128 figure, so its
// workgroup has one wave per SIMD (up to 512 registers each) instead of two.
__host__ __device__ constexpr int max_waves(int head_dim) { return head_dim == 256 ? 4 : kMaxWaves; }
constexpr int kMergeThreads = 256;
constexpr int kMaxLdsBytes = 160 * 1024;  // LDS per CU on gfx950
constexpr int kMaxCols = 16;              // MFMA columns: query tokens x heads of a kv head

struct LaunchArgs {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  const int32_t* bt;
  const int32_t* lens;
  uint16_t* out;
  float* ws_acc;      // [slots, hgs, nq * group, head_dim] partial accumulators
  float* ws_ml;       // [slots, hgs, nq * group, 2] partial (max in log2 units, sum)
  int32_t* ws_pref;   // [batch + 1] steps prefix, then [grid] split list, written by the attention kernel
  int32_t* ws_cnt;    // [grid] arrival counters of the fused merge, zero between calls
  int batch, hq, hkv, group, head_dim, page_shift, num_pages, maxp;
  int hgs;            // kv heads per workgroup (a divisor of hkv, at most max_waves(head_dim))
  int waves;          // waves per workgroup: hgs x step phases
  int grid;           // workgroups of the attention kernel
  int min_steps;      // fewest 32-token steps per wave
  float scale;
  int nq;      // query tokens per sequence (causal among them)
  int window;  // sliding window in tokens, 0 = none
  int valu_cols = 0;  // 0: products on the matrix cores; 4 or 8: vector-ALU variant for that many columns
  bool fused = false; // split sequences merged by their last workgroup (no merge kernel)
  // > 0: the fixed split of small calls -- workgroup w takes chunk w % chunks
  // (chunk_steps 32-token steps) of (sequence, kv-head group) w / chunks;
  // grid = batch x (hkv / hgs) x chunks and merge_fixed_kernel merges
  int chunks = 0;
  int chunk_steps = 0;
  // stream-K only: the partial of a workgroup's first piece is kept in LDS
  // and written after its last piece (the launch adds attn_stash_lds_bytes)
  bool stash = false;
};

// The fused merge is planned when the most partial data one sequence can
// have (grid x kv heads per workgroup x columns x head_dim fp32) is at most
// this, so one workgroup reads it in about one memory round trip.
constexpr int64_t kFusedMergeBytes = 128 * 1024;
constexpr int kMaxFusedGrid = 4096;  // arrival counters a workspace holds

hipError_t launch_attn_kernel(const LaunchArgs& a, hipStream_t st);
// Device address of the fixed scratch of the no-allocation entry point on
// device `dev` (which must be current); taken once per device.
constexpr int kMaxDevices = 64;
hipError_t noalloc_scratch(int dev, void** ptr);
hipError_t launch_merge_kernel(const LaunchArgs& a, hipStream_t st);
size_t attn_lds_bytes(int head_dim, int batch, int waves, bool valu = false);
// LDS of an attention launch with the first-piece stash: hgs kv heads x cols
// columns x (head_dim + 4) floats after attn_lds_bytes.
size_t attn_stash_lds_bytes(int head_dim, int batch, int waves, int hgs, int cols, bool valu = false);

}  // namespace pda
