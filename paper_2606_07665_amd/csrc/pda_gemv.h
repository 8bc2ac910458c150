// Internal interface of the decode GEMV kernels (not part of the public ABI).
#pragma once
#include <hip/hip_runtime.h>
#include <cstdint>

namespace pda {

constexpr int kGemvWaves = 4;                   // waves per GEMV workgroup, splitting each segment's k tiles
constexpr int kGemvThreads = 64 * kGemvWaves;
constexpr int kGemvBlocksPerCu = 3;
// Workgroups of gemv_kernel<nbt, r> resident per CU (one wave of each per
// SIMD), set by the kernel's registers: the three- and four-column-tile
// kernels with deep chunks or row groups would take more than 256 registers
// a wave unless held to two waves per SIMD (their launch bounds); the others
// need at most 168, so three fit.
__host__ __device__ constexpr int gemv_blocks_per_cu(int nbt, int r) {
  return (nbt == 3 || nbt * r >= 9) ? 2 : kGemvBlocksPerCu;
}
// Waves per SIMD the launch bounds ask for: only the heavy kernels need it.
__host__ __device__ constexpr int gemv_min_waves_per_simd(int nbt, int r) {
  return gemv_blocks_per_cu(nbt, r) == 2 ? 2 : 1;
}
constexpr int kGemvMinTiles = 4;                // fewest k tiles per wave (on average)
constexpr int kGemvGroupedUnits = 8;            // fewest units per workgroup to group row tiles of one batch tile
// Thin-GEMM form (batches of more than 16): kXWaves waves per workgroup, one
// row tile each, activations staged in LDS kXChunk k tiles at a time.
constexpr int kXWaves = 8;
constexpr int kXBlocksPerCu = 1;  // one workgroup per CU: fewer workgroups per row group, smaller partials
// Measured on batch 64 (3072..8192 square and 3072 x 5120 weights): chunks
// of 4 k tiles with one chunk in flight ran as fast as or faster than chunks
// of 2 or 8 and than two or three chunks of weights in flight.
constexpr int kXChunk = 4;        // k tiles per chunk
constexpr int kXDepth = 1;        // chunks of weights in flight ahead of the one computing
constexpr int kXRing = kXDepth + 1;
constexpr int kXRowBytes = kXChunk * 64 + 16;  // one activation row of a chunk in LDS (padded)
// s_waitcnt for a chunk's x and weights: with weights two or more chunks
// ahead, only the kXChunk weight loads issued after the chunk's x may still
// be in flight; with one, nothing
constexpr int kWaitVmcntWeights = kXDepth > 1 ? (0x0F70 | (kXChunk & 15) | ((kXChunk >> 4) << 14)) : 0x0F70;
__host__ __device__ constexpr int gemv_xlds_lds_bytes(int nbt) { return kXRing * nbt * 16 * kXRowBytes; }
constexpr int kGemvMaxSlots = 16;               // most workgroups sharing one row group
constexpr int kTileRows = 16;                   // rows of W per MFMA tile
constexpr int kTileK = 32;                      // k per MFMA tile
constexpr int kMaxGemvBatch = 256;              // sequences: sixteen 16-column tiles
// Batches above this run only in the thin-GEMM forms (gemv_xlds_kernel with
// 8 column tiles, gemv_thin_kernel with 16, both with row groups of 8
// tiles), which need the rows in groups of 128.
constexpr int kMaxGemvBatchAnyRows = 64;
constexpr int kPackThreads = 256;

// y[b, n] = sum_k x[b, k] W[n, k] over a packed W (see launch_pack), as
// fp32 partials: a work unit is one 32-k tile of a group of `group`
// consecutive 16-row tiles; part[g][j][i][b][16] (tile-major) or
// part[g][j][b][i][16] (sequence-major) holds the contribution of the j-th
// workgroup that touched row group g, for its tile i and sequence b.
// Tile-major partials are written as contiguous 1 KB rows; sequence-major
// ones keep a sequence's rows of a group together (group x 64 bytes), which
// the o_proj epilogue, one workgroup per sequence, reads as whole lines.
// GemvPlan says how the waves split the work.
struct GemvPlan {
  bool xlds;    // thin-GEMM form (gemv_xlds_kernel, kXWaves waves) instead of gemv_kernel
  bool seq_major = false;  // partial layout (see above)
  int grid;     // workgroups
  int slots;    // partial slots per row group (an upper bound)
  int group;    // 16-row tiles per work unit (x fragments are reused across them)
  int64_t blocks, units;
  int kt_count;
};

// seq_major: the caller's epilogue reads sequence-major partials better; the
// plan takes that layout except in gemv_thin_kernel, whose tile-major
// stores it would spread out.
GemvPlan plan_gemv(int batch, int n, int k, int num_cus, bool seq_major = false);
int64_t gemv_partial_floats(const GemvPlan& p, int batch, int n);

struct GemvArgs {
  const uint16_t* x;   // bf16 [batch, k]
  const uint16_t* wp;  // packed bf16 [n, k]
  float* part;         // fp32 partials, gemv_partial_floats() of them
  int batch, n, k;
  GemvPlan plan;
};

struct PreludeArgs {
  const float* part;         // GEMV partials of y [batch, (hq + 2 hkv) * d]
  GemvPlan plan;
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
  // theta^(-2 * 2^k / rotary_dim) for k = 0..7, in fp64 from the host: the
  // frequency theta^(-2i/rotary_dim) of pair i (i < 128) is the product of
  // those for the set bits of i
  double freq_pow2[8];
  float eps;
};

// o_proj epilogue, two passes over (sequence, chunk of kOProjChunk features):
// z = y + residual and the chunk's sum of z^2, then h = RMSNorm(z) * w once
// every chunk's sum is known.
constexpr int kOProjChunk = 256;                // features per workgroup (one per thread)
constexpr int kMaxOProjHidden = 32768;

struct OProjArgs {
  const float* part;          // GEMV partials of y [batch, hidden]
  GemvPlan plan;
  const uint16_t* residual;   // bf16 [batch, hidden]
  const uint16_t* norm_w;     // bf16 [hidden]
  uint16_t* residual_out;     // bf16 [batch, hidden] (may be residual itself)
  uint16_t* normed_out;       // bf16 [batch, hidden]
  float* z;                   // fp32 [batch, hidden] scratch
  float* chunk_ss;            // fp32 [batch, chunks] scratch
  int batch, hidden;
  float eps;
};

__host__ __device__ inline int oproj_chunks(int hidden) { return (hidden + kOProjChunk - 1) / kOProjChunk; }

// The o_proj epilogue runs as one kernel when the hidden size allows: one
// workgroup of kOProjOneThreads per sequence holds all of its z in
// registers (at most kOProjOneFeatures per thread), so the norm needs no
// second pass.  Measured faster than or as fast as the two passes at
// batches 1, 4, 16, 64 and 256; larger hidden sizes keep the two passes.
constexpr int kOProjOneThreads = 1024;
constexpr int kOProjOneFeatures = 8;
constexpr int kOProjOneMaxBatch = 256;
__host__ __device__ inline bool oproj_one_kernel(int batch, int hidden) {
  return batch <= kOProjOneMaxBatch && hidden <= kOProjOneThreads * kOProjOneFeatures;
}

hipError_t launch_pack(const uint16_t* w, uint16_t* wp, int n, int k, hipStream_t st);
hipError_t launch_oproj_epilogue(const OProjArgs& a, hipStream_t st);
hipError_t launch_gemv(const GemvArgs& a, hipStream_t st);
hipError_t launch_prelude_epilogue(const PreludeArgs& a, hipStream_t st);

}  // namespace pda
