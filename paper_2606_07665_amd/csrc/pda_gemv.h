// Internal interface of the decode GEMV kernels (not part of the public ABI).
#pragma once
#include <hip/hip_runtime.h>
#include <cstdint>

namespace pda {

constexpr int kGemvWaves = 8;                   // waves per GEMV workgroup, splitting K
constexpr int kGemvThreads = 64 * kGemvWaves;
constexpr int kTileRows = 16;                   // rows of W per MFMA tile
constexpr int kTileK = 32;                      // k per MFMA tile
constexpr int kMaxGemvBatch = 64;               // sequences: four 16-column tiles
constexpr int kPackThreads = 256;

// y[b, n] = sum_k x[b, k] W[n, k] over a packed W (see launch_pack), fp32 out.
struct GemvArgs {
  const uint16_t* x;   // bf16 [batch, k]
  const uint16_t* wp;  // packed bf16 [n, k]
  float* y;            // fp32 [batch, n]
  int batch, n, k;
};

struct PreludeArgs {
  const float* y;            // fp32 [batch, (hq + 2 hkv) * d]
  const uint16_t* bias;      // bf16 [(hq + 2 hkv) * d] or null
  const uint16_t* q_norm;    // bf16 [d] or null
  const uint16_t* k_norm;    // bf16 [d] or null
  const int32_t* lens;       // [batch]
  uint16_t* q_out;           // bf16 [batch, hq, d]
  uint16_t* k_out;           // bf16 [batch, hkv, d] or null
  uint16_t* v_out;
  uint16_t* k_cache;         // bf16 [num_pages, page, hkv, d] or null (no append)
  uint16_t* v_cache;
  const int32_t* bt;         // [batch, maxp]
  int page_shift, num_pages, maxp;
  int batch, hq, hkv, d, rotary_dim, interleaved;
  float theta, eps;
};

hipError_t launch_pack(const uint16_t* w, uint16_t* wp, int n, int k, hipStream_t st);
hipError_t launch_gemv(const GemvArgs& a, hipStream_t st);
hipError_t launch_prelude_epilogue(const PreludeArgs& a, hipStream_t st);

}  // namespace pda
