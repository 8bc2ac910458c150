// Internal interface between the C-ABI host code and the HIP kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace pda {

constexpr int kBlockThreads = 256;            // 4 independent wave64 workers
constexpr int kWavesPerBlock = kBlockThreads / 64;
constexpr int kStep = 32;                     // tokens per pipeline step of a wave
constexpr int kMaxLdsBytes = 160 * 1024;      // LDS per CU on gfx950

struct LaunchArgs {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  const int32_t* bt;
  const int32_t* lens;
  uint16_t* out;
  float* ws_acc;      // [slots, group, head_dim] partial accumulators
  float* ws_ml;       // [slots, group, 2] partial (max in log2 units, sum)
  int32_t* ws_cnt;    // [batch * hkv] arrival counters, zero between calls
  int batch, hq, hkv, group, head_dim, page_shift, num_pages, maxp;
  int grid;           // workgroups of the kernel
  int min_steps;      // fewest 32-token steps per wave of a workgroup
  float scale;
};

hipError_t launch_split_kernel(const LaunchArgs& a, hipStream_t st);
size_t split_lds_bytes(int head_dim, int batch);

}  // namespace pda
