// Decode GEMV, the attention prelude and the output projection for MI355X
// (gfx950, CDNA4, wave64).
//
// What is computed: the paper's kernel family (i), the attention prelude
// (Method, "Principle-Driven LLM Kernel Generator"): the QKV projection of
// the new token's hidden state, then per-head RMSNorm of q and k (when the
// model has it) and the rotary position embedding of q and k.  Its template
// GEMV (Method, "CUDA Code Generator") reads [N, K] weight rows with 128-bit
// loads and reduces across lanes; on CDNA4 the same bandwidth-bound
// product is laid out differently:
//
//  * Weights are packed once into the matrix cores' operand order: a tile of
//    16 rows x 32 k is 1 KB, and lane l of a wave holds row l % 16, k
//    8 (l / 16) .. +7 of it.  Every weight load of the GEMV is then one
//    contiguous 1 KB wave access that feeds v_mfma_f32_16x16x32_bf16
//    directly, with no LDS staging and no lane shuffles.
//  * The batch forms the MFMA's B columns in 16-column tiles (up to four in
//    gemv_kernel, up to sixteen -- 256 sequences -- in the thin-GEMM form);
//    x rows past the batch read as zeros through the buffer descriptor's
//    size.
//  * Stream-K over (row group, 32-k tile) units: every workgroup of a grid
//    sized to the device streams the same number of packed weight tiles,
//    whatever the shape, so no half-empty last round of workgroups.  The
//    waves of a workgroup split its k tiles and add their accumulators in
//    LDS; the workgroup leaves one fp32 partial per row group it touched and
//    the epilogue adds a group's partials in workgroup order.
//  * The epilogue (partial sums, bias, RMSNorm, rotation, bf16 rounding, and
//    optionally the KV append into the page slot) runs per (sequence, head):
//    a head's norm and its rotation pairs need all of its rows, which no
//    single wave of the GEMV holds.
//
// The output projection after attention (kernel family (v): o_proj GEMV +
// residual add + the RMSNorm that follows) runs on the same GEMV; its
// epilogue works in two passes over (sequence, chunk of features), since the
// norm spans all hidden features of a sequence.
#include "pda_gemv.h"

#include <atomic>
#include <cstdlib>

namespace pda {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));

constexpr int kBufferDword3 = 0x00020000;  // raw 32-bit buffer format
constexpr int kCachePolicyNT = 2;          // non-temporal: weights are read once

__device__ __forceinline__ int uniform(int x) { return __builtin_amdgcn_readfirstlane(x); }

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  const uint64_t a = reinterpret_cast<uint64_t>(base);
  const uint32_t lo = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(a));
  const uint32_t hi = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(a >> 32));
  void* ub = reinterpret_cast<void*>((static_cast<uint64_t>(hi) << 32) | lo);
  return __builtin_amdgcn_make_buffer_rsrc(ub, 0, static_cast<int>(__builtin_amdgcn_readfirstlane(bytes)),
                                           kBufferDword3);
}

// Packed layout: tile (t, kt) of rows 16t .. 16t+15 and k 32kt .. 32kt+31 is
// stored at element (t * (k / 32) + kt) * 512; inside it, 16-byte chunk l
// holds W[16t + l % 16][32kt + 8 (l / 16) .. +7].  One thread per chunk.
__global__ __launch_bounds__(kPackThreads) void pack_kernel(const uint16_t* __restrict__ w,
                                                            uint16_t* __restrict__ wp, int n, int k) {
  const int64_t chunk = static_cast<int64_t>(blockIdx.x) * kPackThreads + threadIdx.x;
  const int64_t chunks = static_cast<int64_t>(n) * k / 8;
  if (chunk >= chunks) return;
  const int kt_count = k / kTileK;
  const int64_t tile = chunk / 64;
  const int l = static_cast<int>(chunk % 64);
  const int64_t t = tile / kt_count;
  const int kt = static_cast<int>(tile % kt_count);
  const int64_t row = t * kTileRows + (l & 15);
  const int64_t col = static_cast<int64_t>(kt) * kTileK + 8 * (l >> 4);
  *reinterpret_cast<u32x4*>(wp + chunk * 8) = *reinterpret_cast<const u32x4*>(w + row * k + col);
}

// Stream-K GEMV: the flattened space of (row group g, 32-k tile) units is
// cut into equal contiguous ranges, one per workgroup, so every workgroup
// streams the same number of packed weight tiles whatever the matrix shape.
// A row group is kR consecutive 16-row tiles: each x fragment a wave loads
// feeds kR MFMAs, which keeps x reads (L2) at or below the weight reads
// (HBM) when the batch spans several 16-column tiles, and cuts them 4x
// within one tile of more than 4 sequences.  Inside a workgroup
// the 4 waves split each group segment's k tiles into contiguous quarters
// and add their accumulators in LDS; the workgroup then writes one partial
// (kR tiles x batch, fp32) per row group its range touches, into slot
// j = workgroup - first_workgroup(g) of that group, and the epilogue sums a
// group's slots in order (deterministic).
template <int kNBT, int kR>
__global__ __launch_bounds__(kGemvThreads, gemv_min_waves_per_simd(kNBT, kR)) void gemv_kernel(
    const uint16_t* __restrict__ x, const uint16_t* __restrict__ wp, float* __restrict__ part, int batch, int n,
    int k, int slots, int seq_major) {
  __shared__ f32x4 red[kGemvWaves][kR * kNBT][64];
  const int lane = threadIdx.x & 63;
  const int wv = uniform(threadIdx.x >> 6);
  const int64_t blocks = gridDim.x;
  const int64_t blk = blockIdx.x;
  const int kt_count = k / kTileK;
  const int64_t units = static_cast<int64_t>(n / (kTileRows * kR)) * kt_count;
  int64_t u = blk * units / blocks;
  const int64_t u_end = (blk + 1) * units / blocks;

  // x rows at or past the batch fall outside the descriptor and read as zeros
  const __amdgpu_buffer_rsrc_t rx = make_rsrc(x, static_cast<uint32_t>(batch) * k * 2u);
  const int r = lane & 15;
  const int g4 = lane >> 4;
  int xrow[kNBT];
#pragma unroll
  for (int bt = 0; bt < kNBT; ++bt) xrow[bt] = ((16 * bt + r) * k + 8 * g4) * 2;

  while (u < u_end) {
    const int g = static_cast<int>(u / kt_count);
    const int64_t seg_end = u_end < static_cast<int64_t>(g + 1) * kt_count ? u_end
                                                                           : static_cast<int64_t>(g + 1) * kt_count;
    const int seg = static_cast<int>(seg_end - u);
    // this wave's quarter of the segment: k tiles [kt0, kt0 + per)
    const int lo = wv * seg / kGemvWaves;
    const int per = (wv + 1) * seg / kGemvWaves - lo;
    const int kt0 = static_cast<int>(u - static_cast<int64_t>(g) * kt_count) + lo;
    const uint16_t* wbase = wp + (static_cast<int64_t>(g) * kR * kt_count + kt0) * (kTileRows * kTileK);
    __amdgpu_buffer_rsrc_t rw[kR];
#pragma unroll
    for (int i = 0; i < kR; ++i)  // k tiles past the quarter read as zeros (outside the descriptor)
      rw[i] = make_rsrc(wbase + static_cast<int64_t>(i) * kt_count * (kTileRows * kTileK),
                        static_cast<uint32_t>(per) * 1024u);

    f32x4 acc[kR][kNBT];
#pragma unroll
    for (int i = 0; i < kR; ++i)
#pragma unroll
      for (int bt = 0; bt < kNBT; ++bt) acc[i][bt] = f32x4{0.f, 0.f, 0.f, 0.f};
    // k tiles in chunks, the next chunk's loads in flight while the current
    // chunk's MFMAs run
    constexpr int kChunk = kNBT * kR >= 4 ? 2 : (kNBT == 1 ? 8 : 4);
    u32x4 wa[2][kChunk][kR];
    u32x4 xb[2][kChunk][kNBT];
    auto load = [&](int buf, int j0) {
#pragma unroll
      for (int j = 0; j < kChunk; ++j) {
#pragma unroll
        for (int i = 0; i < kR; ++i)
          wa[buf][j][i] = __builtin_amdgcn_raw_buffer_load_b128(rw[i], (j0 + j) * 1024 + 16 * lane, 0, kCachePolicyNT);
        const bool in = j0 + j < per;
#pragma unroll
        for (int bt = 0; bt < kNBT; ++bt)
          xb[buf][j][bt] = in ? __builtin_amdgcn_raw_buffer_load_b128(rx, xrow[bt] + (kt0 + j0 + j) * kTileK * 2, 0, 0)
                              : u32x4{0u, 0u, 0u, 0u};
      }
    };
    auto mma = [&](int buf) {
#pragma unroll
      for (int j = 0; j < kChunk; ++j)
#pragma unroll
        for (int i = 0; i < kR; ++i)
#pragma unroll
          for (int bt = 0; bt < kNBT; ++bt)
            acc[i][bt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, wa[buf][j][i]),
                                                                 __builtin_bit_cast(bf16x8, xb[buf][j][bt]),
                                                                 acc[i][bt], 0, 0, 0);
    };
    const int chunks = (per + kChunk - 1) / kChunk;
    if (chunks > 0) {
      load(0, 0);
      int c = 0;
      for (; c + 2 <= chunks; c += 2) {
        load(1, (c + 1) * kChunk);
        mma(0);
        if (c + 2 < chunks) load(0, (c + 2) * kChunk);
        mma(1);
      }
      if (c < chunks) mma(0);
    }

    // the 4 waves' accumulators meet in LDS; wave wv adds and stores the
    // (tile, column tile) pairs wv, wv + 4, ...
#pragma unroll
    for (int i = 0; i < kR; ++i)
#pragma unroll
      for (int bt = 0; bt < kNBT; ++bt) red[wv][i * kNBT + bt][lane] = acc[i][bt];
    __syncthreads();
    // C layout: lane holds rows 4 (l / 16) + i, column l % 16 of its tile
    const int64_t first = (static_cast<int64_t>(g) * kt_count * blocks + blocks - 1) / units;  // first block of g
    float* slot = part + (static_cast<int64_t>(g) * slots + (blk - first)) * kR * batch * kTileRows;
    for (int p = wv; p < kR * kNBT; p += kGemvWaves) {
      const int i = p / kNBT;
      const int bt = p - i * kNBT;
      f32x4 sum = red[0][p][lane];
#pragma unroll
      for (int w2 = 1; w2 < kGemvWaves; ++w2) sum += red[w2][p][lane];
      const int b = 16 * bt + r;
      const int row = seq_major ? b * kR + i : i * batch + b;
      if (b < batch) *reinterpret_cast<f32x4*>(slot + row * kTileRows + 4 * g4) = sum;
    }
    __syncthreads();  // red is rewritten by the next segment
    u = seg_end;
  }
}

// Thin-GEMM form of the same stream-K GEMV for batches of more than 16
// sequences.  A workgroup of kXWaves waves works on row groups of kXWaves
// row tiles, wave w on tile w of the group, over the group's k range in
// chunks of kXChunk k tiles: the chunk's activations (batch x kXChunk x 32
// bf16) are loaded once per workgroup with row-contiguous reads and staged
// in LDS, where every wave reads its B fragments; the weights come straight
// from the packed tiles into registers, kXDepth chunks ahead.  Compared with
// gemv_kernel (x fragments loaded per wave, 16 rows x 64 bytes per load,
// reused across the group's row tiles in registers), the x reads from L2
// halve and are contiguous, and no cross-wave reduction is needed since each
// wave owns its rows.  Partials and their layout are gemv_kernel's (group =
// kXWaves tiles), so the epilogues are shared.
template <int kNBT>
__global__ __launch_bounds__(kXWaves * 64, 1) void gemv_xlds_kernel(
    const uint16_t* __restrict__ x, const uint16_t* __restrict__ wp, float* __restrict__ part, int batch, int n,
    int k, int slots, int seq_major) {
  extern __shared__ __align__(16) unsigned char xs[];  // [kXRing][kNBT * 16 rows][kXRowBytes]
  constexpr int kRows = kNBT * kTileRows;
  constexpr int kBuf = kRows * kXRowBytes;
  constexpr int kRowPieces = kXChunk * kTileK / 8;                       // 16-byte pieces per row and chunk
  constexpr int kPieces = kRows * kRowPieces;
  constexpr int kPer = (kPieces + kXWaves * 64 - 1) / (kXWaves * 64);  // per thread
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wv = uniform(tid >> 6);
  const int64_t blocks = gridDim.x;
  const int64_t blk = blockIdx.x;
  const int kt_count = k / kTileK;
  const int64_t units = static_cast<int64_t>(n / (kTileRows * kXWaves)) * kt_count;
  int64_t u = blk * units / blocks;
  const int64_t u_end = (blk + 1) * units / blocks;
  // x rows at or past the batch fall outside the descriptor and read as zeros
  const __amdgpu_buffer_rsrc_t rx = make_rsrc(x, static_cast<uint32_t>(batch) * k * 2u);
  const int r = lane & 15;
  const int g4 = lane >> 4;
  constexpr uint32_t kOutside = 0x80000000u;  // a buffer offset past any descriptor: reads zero

  while (u < u_end) {
    const int g = static_cast<int>(u / kt_count);
    const int64_t seg_end = u_end < static_cast<int64_t>(g + 1) * kt_count ? u_end
                                                                           : static_cast<int64_t>(g + 1) * kt_count;
    const int kt_a = static_cast<int>(u - static_cast<int64_t>(g) * kt_count);
    const int seg = static_cast<int>(seg_end - u);
    const int nch = (seg + kXChunk - 1) / kXChunk;
    // this wave's row tile over the segment; k tiles past it read as zeros
    const uint16_t* wbase = wp + ((static_cast<int64_t>(g) * kXWaves + wv) * kt_count + kt_a) * (kTileRows * kTileK);
    const __amdgpu_buffer_rsrc_t rw = make_rsrc(wbase, static_cast<uint32_t>(seg) * 1024u);

    f32x4 acc[kNBT];
#pragma unroll
    for (int bt = 0; bt < kNBT; ++bt) acc[bt] = f32x4{0.f, 0.f, 0.f, 0.f};
    u32x4 wa[kXRing][kXChunk];
    u32x4 xr[kPer];
    // chunks past the segment load nothing (zero-size reads), so every
    // iteration issues the same loads and the waits are one count
    auto load_w = [&](int buf, int c) {
#pragma unroll
      for (int j = 0; j < kXChunk; ++j)
        wa[buf][j] = __builtin_amdgcn_raw_buffer_load_b128(rw, (c * kXChunk + j) * 1024 + 16 * lane, 0, kCachePolicyNT);
    };
    // piece q: row q / kRowPieces, 16 bytes at k 8 (q % kRowPieces) of the chunk
    auto load_x = [&](int c) {
#pragma unroll
      for (int i = 0; i < kPer; ++i) {
        const int q = tid + i * kXWaves * 64;
        const int row = q / kRowPieces;
        const int kk = c * kXChunk * kTileK + 8 * (q % kRowPieces);  // k within the segment
        const bool live = q < kPieces && kk < seg * kTileK;
        const uint32_t off = live ? static_cast<uint32_t>((row * k + kt_a * kTileK + kk) * 2) : kOutside;
        xr[i] = __builtin_amdgcn_raw_buffer_load_b128(rx, off, 0, 0);
      }
    };
    auto store_x = [&](int buf) {
#pragma unroll
      for (int i = 0; i < kPer; ++i) {
        const int q = tid + i * kXWaves * 64;
        if (q < kPieces)
          *reinterpret_cast<u32x4*>(xs + buf * kBuf + (q / kRowPieces) * kXRowBytes + 16 * (q % kRowPieces)) = xr[i];
      }
    };
    auto mma = [&](int buf) {
#pragma unroll
      for (int j = 0; j < kXChunk; ++j) {
#pragma unroll
        for (int bt = 0; bt < kNBT; ++bt) {
          const u32x4 b = *reinterpret_cast<const u32x4*>(xs + buf * kBuf + (16 * bt + r) * kXRowBytes + 64 * j + 16 * g4);
          acc[bt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, wa[buf][j]),
                                                            __builtin_bit_cast(bf16x8, b), acc[bt], 0, 0, 0);
        }
      }
    };
    // x of chunk c + 1 and the weights of chunk c + kXDepth are in flight
    // while chunk c computes; x goes through a ring of kXRing LDS buffers,
    // so one barrier per chunk orders its writes after the last reads
    load_x(0);
#pragma unroll
    for (int d = 0; d < kXDepth; ++d) load_w(d, d);
    for (int c0 = 0; c0 < nch; c0 += kXRing) {
#pragma unroll
      for (int sl = 0; sl < kXRing; ++sl) {
        const int c = c0 + sl;
        if (c < nch) {
          // everything but the weights issued after x of chunk c has arrived
          __builtin_amdgcn_s_waitcnt(kWaitVmcntWeights);
          store_x(sl);
          load_x(c + 1);
          load_w((sl + kXDepth) % kXRing, c + kXDepth);
          __syncthreads();
          mma(sl);
        }
      }
    }
    // this wave's rows of the group: one partial per (workgroup, group)
    const int64_t first = (static_cast<int64_t>(g) * kt_count * blocks + blocks - 1) / units;  // first block of g
    float* slot = part + (static_cast<int64_t>(g) * slots + (blk - first)) * kXWaves * batch * kTileRows;
#pragma unroll
    for (int bt = 0; bt < kNBT; ++bt) {
      const int b = 16 * bt + r;
      const int row = seq_major ? b * kXWaves + wv : wv * batch + b;
      if (b < batch) *reinterpret_cast<f32x4*>(slot + row * kTileRows + 4 * g4) = acc[bt];
    }
    __builtin_amdgcn_s_waitcnt(0x0F70);  // the loads issued past the segment
    __syncthreads();                     // the LDS buffers are rewritten by the next segment
    u = seg_end;
  }
}

// Thin-GEMM form for the largest batches, with the activations copied
// straight into LDS.  The B fragments of a chunk (kC k tiles x kNBT column
// tiles, 1 KB each) are fetched by the workgroup's waves with buffer loads
// that write LDS directly (no registers, no LDS store instructions): lane l
// of such a load fetches x[16 bt + l % 16][32 kt + 8 (l / 16) .. +7], so each
// fragment lands in LDS in exactly the order the matrix cores read it and
// every LDS read of a fragment is one contiguous, conflict-free 1 KB wave
// access.  Weights come from the packed tiles into registers, kR row tiles
// per wave, so each B fragment read from LDS feeds kR MFMAs: at 256
// sequences a wave of gemv_xlds_kernel reads 16 KB of fragments from LDS per
// 1 KB weight tile, this form 8 KB.  Activations and weights are both kD
// chunks ahead through a ring of kD + 1 stages, with one barrier per chunk.
// The workgroup's range of (row group, k tile) units is walked as one
// stream: where it passes into the next row group the accumulators are
// written out as that group's partial and cleared, while the loads keep
// flowing.  Partials and their layout are gemv_kernel's (group = kW kR row
// tiles).
template <int kNBT, int kW, int kR, int kC, int kD>
__global__ __launch_bounds__(kW * 64, 1) void gemv_thin_kernel(const uint16_t* __restrict__ x,
                                                               const uint16_t* __restrict__ wp,
                                                               float* __restrict__ part, int batch, int n, int k,
                                                               int slots) {
  extern __shared__ __align__(1024) unsigned char xs[];  // [kD + 1][kC][kNBT] fragments of 1 KB
  constexpr int kGroup = kW * kR;
  constexpr int kFrags = kC * kNBT;
  static_assert(kFrags % kW == 0, "every wave copies the same number of fragments");
  constexpr int kDma = kFrags / kW;
  constexpr int kStages = kD + 1;
  constexpr int kLoads = kDma + kC * kR;  // vector memory instructions per wave and chunk
  static_assert(kD >= 2, "the next chunk's loads are waited for while later ones stay in flight");
  constexpr int kAheadFirst = (kD - 1) * kLoads;  // after chunk 0's loads
  constexpr int kAheadNext = (kD - 2) * kLoads;   // after chunk c + 1's loads, at chunk c
  static_assert(kAheadFirst < 64, "vmcnt holds at most 63");
  // vmcnt(n) with expcnt and lgkmcnt not waited for / with lgkmcnt(0)
  constexpr int kWaitFirst = 0x0F70 | (kAheadFirst & 15) | ((kAheadFirst >> 4) << 14);
  constexpr int kWaitNext = 0x0070 | (kAheadNext & 15) | ((kAheadNext >> 4) << 14);
  constexpr uint32_t kOutside = 0x80000000u;  // past any descriptor of x: reads zero
  const int lane = threadIdx.x & 63;
  const int wv = uniform(threadIdx.x >> 6);
  const int64_t blocks = gridDim.x;
  const int64_t blk = blockIdx.x;
  const int kt_count = k / kTileK;
  const int64_t units = static_cast<int64_t>(n / (kTileRows * kGroup)) * kt_count;
  const int64_t u0 = blk * units / blocks;
  const int64_t u1 = (blk + 1) * units / blocks;
  const int nch = static_cast<int>((u1 - u0 + kC - 1) / kC);
  // x rows at or past the batch fall outside the descriptor and read as zeros
  const __amdgpu_buffer_rsrc_t rx = make_rsrc(x, static_cast<uint32_t>(batch) * k * 2u);
  const uint32_t xlane = static_cast<uint32_t>(((lane & 15) * k + 8 * (lane >> 4)) * 2);

  // load stream: the (group, k tile) of the next unit to fetch
  int lg = static_cast<int>(u0 / kt_count);
  int lkt = static_cast<int>(u0 - static_cast<int64_t>(lg) * kt_count);
  int64_t lu = u0;
  u32x4 wa[kStages][kC][kR];
  auto issue = [&](int stage) __attribute__((always_inline)) {
    int gj[kC], ktj[kC];
    bool live[kC];
#pragma unroll
    for (int j = 0; j < kC; ++j) {
      gj[j] = lg;
      ktj[j] = lkt;
      live[j] = lu < u1;
      ++lu;
      if (++lkt == kt_count) {
        lkt = 0;
        ++lg;
      }
    }
#pragma unroll
    for (int d = 0; d < kDma; ++d) {
      const int f = wv * kDma + d;  // fragment (j, bt) of the chunk
      const int j = f / kNBT;
      const int bt = f - j * kNBT;
      const uint32_t off = live[j] ? xlane + static_cast<uint32_t>((16 * bt * k + ktj[j] * kTileK) * 2) : kOutside;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rx, (__attribute__((address_space(3))) void*)(xs + (stage * kFrags + f) * 1024),
                                               16, off, 0, 0, 0);
    }
#pragma unroll
    for (int j = 0; j < kC; ++j) {
#pragma unroll
      for (int r = 0; r < kR; ++r) {
        const int64_t tile = static_cast<int64_t>(gj[j]) * kGroup + wv * kR + r;
        const __amdgpu_buffer_rsrc_t rw =
            make_rsrc(wp + (tile * kt_count + ktj[j]) * (kTileRows * kTileK), live[j] ? 1024u : 0u);
        wa[stage][j][r] = __builtin_amdgcn_raw_buffer_load_b128(rw, 16 * lane, 0, kCachePolicyNT);
      }
    }
  };

  f32x4 acc[kR][kNBT];
#pragma unroll
  for (int r = 0; r < kR; ++r)
#pragma unroll
    for (int bt = 0; bt < kNBT; ++bt) acc[r][bt] = f32x4{0.f, 0.f, 0.f, 0.f};
  const int r16 = lane & 15;
  const int g4 = lane >> 4;
  // this wave's rows of group g as the workgroup's partial of g, then cleared
  auto flush = [&](int g) __attribute__((always_inline)) {
    const int64_t first = (static_cast<int64_t>(g) * kt_count * blocks + blocks - 1) / units;  // first block of g
    float* slot = part + (static_cast<int64_t>(g) * slots + (blk - first)) * kGroup * batch * kTileRows;
#pragma unroll
    for (int r = 0; r < kR; ++r)
#pragma unroll
      for (int bt = 0; bt < kNBT; ++bt) {
        const int b = 16 * bt + r16;
        if (b < batch) *reinterpret_cast<f32x4*>(slot + ((wv * kR + r) * batch + b) * kTileRows + 4 * g4) = acc[r][bt];
        acc[r][bt] = f32x4{0.f, 0.f, 0.f, 0.f};
      }
  };
  // compute stream: the (group, k tile) of the next unit to accumulate
  int mg = lg;
  int mkt = lkt;
  int64_t mu = u0;
  // B fragments of the chunk being multiplied; each register is refilled
  // with the next chunk's fragment right after the kR MFMAs that read it,
  // so the LDS reads of chunk c + 1 run under the MFMAs of chunk c and no
  // MFMA waits for LDS.  A unit's partial flush comes before its MFMAs.
  u32x4 b[kC][kNBT];
  auto frag = [&](int stage, int j, int bt) __attribute__((always_inline)) {
    return *reinterpret_cast<const u32x4*>(xs + ((stage * kC + j) * kNBT + bt) * 1024 + 16 * lane);
  };
  auto mma = [&](int stage, int next) __attribute__((always_inline)) {
#pragma unroll
    for (int j = 0; j < kC; ++j) {
      if (mu < u1 && mkt == 0 && mu != u0) flush(mg - 1);
      // a chunk past the range holds zeros in LDS and in its weight
      // registers (both read outside their descriptors), so its MFMAs add
      // exact zeros: no branch around them
#pragma unroll
      for (int bt = 0; bt < kNBT; ++bt) {
#pragma unroll
        for (int r = 0; r < kR; ++r)
          acc[r][bt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, wa[stage][j][r]),
                                                               __builtin_bit_cast(bf16x8, b[j][bt]), acc[r][bt], 0, 0, 0);
        b[j][bt] = frag(next, j, bt);
      }
#pragma unroll
      for (int bt = 0; bt < kNBT; ++bt) {
        __builtin_amdgcn_sched_group_barrier(0x008, kR, 0);  // the kR MFMAs of fragment bt
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);   // then its refill
      }
      ++mu;
      if (++mkt == kt_count) {
        mkt = 0;
        ++mg;
      }
    }
  };

  // Chunks past the range load nothing (zero-size reads) and add zeros,
  // so every chunk issues the same loads, the waits are fixed counts, and
  // the ring is walked in whole turns (a range is padded by at most
  // kStages - 1 such chunks): with a branch around each stage the compiler
  // must allow for skipped stages, and it then waited for every load but
  // the newest chunk's before the MFMAs, one chunk of prefetch whatever the
  // depth.  The prologue keeps each chunk's loads in the loop's order
  // (copies, then weights), so the first turn counts like the others.
#pragma unroll
  for (int s = 0; s < kD; ++s) {
    issue(s);
    __builtin_amdgcn_sched_barrier(0);
  }
  // chunk 0 in LDS for every wave, then its fragments into registers
  __builtin_amdgcn_s_waitcnt(kWaitFirst);
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
#pragma unroll
  for (int j = 0; j < kC; ++j)
#pragma unroll
    for (int bt = 0; bt < kNBT; ++bt) b[j][bt] = frag(0, j, bt);
  for (int c0 = 0; c0 < nch; c0 += kStages) {
#pragma unroll
    for (int s = 0; s < kStages; ++s) {
      // At chunk c = c0 + s: this wave's copies and weights of chunk c + 1
      // have landed and its reads of chunk c's fragments are done; after the
      // barrier every wave's copies of chunk c + 1 are in LDS and stage
      // s - 1 (chunk c - 1, read during chunk c - 2) is free for chunk
      // c + kD.  A bare s_barrier, fenced for the compiler only: a workgroup
      // fence would also wait for the copies still in flight into the later
      // stages.
      __builtin_amdgcn_s_waitcnt(kWaitNext);
      asm volatile("" ::: "memory");
      __builtin_amdgcn_s_barrier();
      asm volatile("" ::: "memory");
      issue((s + kD) % kStages);
      mma(s, (s + 1) % kStages);
    }
  }
  if (u1 > u0) {
    // the group of the range's last unit
    const int64_t last = u1 - 1;
    flush(static_cast<int>(last / kt_count));
  }
  __builtin_amdgcn_s_waitcnt(0x0F70);  // copies into LDS still in flight end before the workgroup does
}

// y[b][rows[r]] for kRows rows: for each, the sum in workgroup order of the
// partials of its row group (kSlots >= the plan's slots, the most
// workgroups that touch one group).  All partial counts are worked out
// first, under one uniform branch (32-bit arithmetic when every product
// fits, as on 256 CUs for every supported shape; each 64-bit division is a
// long instruction sequence), then every load is issued unconditionally:
// slots past a group's count re-read its last slot and are dropped by a
// select after the load.  As `j < cnt ? load : 0`, each load sat behind a
// branch of its own and a lane waited for one row's partials before it
// requested the next row's.
template <int kSlots, int kRows>
__device__ __forceinline__ void gemv_rows(const float* __restrict__ part, const GemvPlan& p, int batch, int b,
                                          const int (&rows)[kRows], float (&y)[kRows]) {
  int g[kRows], cnt[kRows];
#pragma unroll
  for (int r = 0; r < kRows; ++r) g[r] = (rows[r] >> 4) / p.group;
  if (((p.units * p.blocks) >> 32) == 0) {
    const uint32_t nb = static_cast<uint32_t>(p.blocks), nu = static_cast<uint32_t>(p.units);
#pragma unroll
    for (int r = 0; r < kRows; ++r) {
      const uint32_t x0 = static_cast<uint32_t>(g[r]) * p.kt_count;
      cnt[r] = static_cast<int>(((x0 + p.kt_count) * nb - 1) / nu - ((x0 + 1) * nb - 1) / nu + 1);
    }
  } else {
#pragma unroll
    for (int r = 0; r < kRows; ++r) {
      const int64_t x0 = static_cast<int64_t>(g[r]) * p.kt_count;
      cnt[r] = static_cast<int>(((x0 + p.kt_count) * p.blocks - 1) / p.units - ((x0 + 1) * p.blocks - 1) / p.units + 1);
    }
  }
  const int64_t slot_floats = static_cast<int64_t>(p.group) * batch * kTileRows;
  float v[kRows][kSlots];
#pragma unroll
  for (int r = 0; r < kRows; ++r) {
    const int i = (rows[r] >> 4) - g[r] * p.group;
    const float* q = part + static_cast<int64_t>(g[r]) * p.slots * slot_floats +
                     (p.seq_major ? static_cast<int64_t>(b) * p.group + i : static_cast<int64_t>(i) * batch + b) *
                         kTileRows +
                     (rows[r] & 15);
#pragma unroll
    for (int j = 0; j < kSlots; ++j) v[r][j] = q[(j < cnt[r] ? j : cnt[r] - 1) * slot_floats];
  }
#pragma unroll
  for (int r = 0; r < kRows; ++r) {
    float s = 0.f;
#pragma unroll
    for (int j = 0; j < kSlots; ++j) s += j < cnt[r] ? v[r][j] : 0.f;
    y[r] = s;
  }
}

// y[b][n .. n+3] for four consecutive rows n (n a multiple of 4, so one
// 16-byte piece of one tile's partial row in every slot): the sum in
// workgroup order of their group's partials, loaded as 16-byte pieces,
// every slot's load issued before any is added.
template <int kSlots>
__device__ __forceinline__ float4 gemv_rows4(const float* __restrict__ part, const GemvPlan& p, int batch, int b,
                                             int n) {
  const int g = (n >> 4) / p.group;
  int cnt;
  if (((p.units * p.blocks) >> 32) == 0) {
    const uint32_t nb = static_cast<uint32_t>(p.blocks), nu = static_cast<uint32_t>(p.units);
    const uint32_t x0 = static_cast<uint32_t>(g) * p.kt_count;
    cnt = static_cast<int>(((x0 + p.kt_count) * nb - 1) / nu - ((x0 + 1) * nb - 1) / nu + 1);
  } else {
    const int64_t x0 = static_cast<int64_t>(g) * p.kt_count;
    cnt = static_cast<int>(((x0 + p.kt_count) * p.blocks - 1) / p.units - ((x0 + 1) * p.blocks - 1) / p.units + 1);
  }
  const int64_t slot_floats = static_cast<int64_t>(p.group) * batch * kTileRows;
  const int i = (n >> 4) - g * p.group;
  const float* q = part + static_cast<int64_t>(g) * p.slots * slot_floats +
                   (p.seq_major ? static_cast<int64_t>(b) * p.group + i : static_cast<int64_t>(i) * batch + b) *
                       kTileRows +
                   (n & 15);
  float4 v[kSlots];
#pragma unroll
  for (int j = 0; j < kSlots; ++j) v[j] = *reinterpret_cast<const float4*>(q + (j < cnt ? j : cnt - 1) * slot_floats);
  float4 y = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
  for (int j = 0; j < kSlots; ++j)
    if (j < cnt) {
      y.x += v[j].x;
      y.y += v[j].y;
      y.z += v[j].z;
      y.w += v[j].w;
    }
  return y;
}

__device__ __forceinline__ float bf16_to_f32(uint16_t h) {
  return __builtin_bit_cast(float, static_cast<uint32_t>(h) << 16);
}

__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  return __builtin_bit_cast(uint16_t, static_cast<__bf16>(f));
}

// One wave per (sequence b, head h) of the projection: h < hq is a q head,
// then hkv k heads, then hkv v heads.  Lane owns elements lane + 64 j.
template <int D, int kSlots>
__global__ __launch_bounds__(64) void prelude_epilogue(PreludeArgs a) {
  constexpr int E = D / 64;
  __shared__ float s[D];
  const int heads = a.hq + 2 * a.hkv;
  const int b = blockIdx.x / heads;
  const int h = blockIdx.x - b * heads;
  const int lane = threadIdx.x;
  const bool is_q = h < a.hq;
  const bool is_k = !is_q && h < a.hq + a.hkv;
  const uint16_t* nw = is_q ? a.q_norm : (is_k ? a.k_norm : nullptr);

  // Everything the wave reads is requested before any of it is used: the
  // length, then (for an append) the page id of the new token's slot, the
  // partials, the bias and the norm weights.
  const int L = a.lens[b];
  const int pos = L > 0 ? L - 1 : 0;
  const bool kv_head = !is_q;
  const int g = kv_head ? (is_k ? h - a.hq : h - a.hq - a.hkv) : 0;
  uint16_t* cache = kv_head ? (is_k ? a.k_cache : a.v_cache) : nullptr;
  int64_t row = 0;
  if (cache) {
    const int max_ctx = a.maxp << a.page_shift;
    const int Lc = L < 0 ? 0 : (L > max_ctx ? max_ctx : L);
    if (Lc == 0) {
      cache = nullptr;  // no token in this slot: nothing to append
    } else {
      const int t = Lc - 1;
      const unsigned raw = static_cast<unsigned>(a.bt[static_cast<int64_t>(b) * a.maxp + (t >> a.page_shift)]);
      const int64_t page = raw < static_cast<unsigned>(a.num_pages) ? raw : a.num_pages - 1;
      row = (((page << a.page_shift) + (t & ((1 << a.page_shift) - 1))) * a.hkv + g) * D;
    }
  }
  // bias and norm weights are loaded whether present or not (from the
  // partials, a valid address, when absent; dropped by a select), so that
  // no load waits behind a branch
  const uint16_t* bias_p = a.bias ? a.bias + h * D : reinterpret_cast<const uint16_t*>(a.part);
  const uint16_t* nw_p = nw ? nw : reinterpret_cast<const uint16_t*>(a.part);
  int rows[E];
  float v[E];
  uint16_t bias_h[E], wn_h[E];
#pragma unroll
  for (int j = 0; j < E; ++j) {
    rows[j] = h * D + lane + 64 * j;
    bias_h[j] = bias_p[lane + 64 * j];
    wn_h[j] = nw_p[lane + 64 * j];
  }
  gemv_rows<kSlots>(a.part, a.plan, a.batch, b, rows, v);
#pragma unroll
  for (int j = 0; j < E; ++j) v[j] += a.bias ? bf16_to_f32(bias_h[j]) : 0.f;
  if (nw) {
    float ss = 0.f;
#pragma unroll
    for (int j = 0; j < E; ++j) ss += v[j] * v[j];
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) ss += __shfl_xor(ss, off);
    const float inv = rsqrtf(ss / D + a.eps);
#pragma unroll
    for (int j = 0; j < E; ++j) v[j] = v[j] * inv * bf16_to_f32(wn_h[j]);
  }
  if ((is_q || is_k) && a.rotary_dim > 0) {
    const int r = a.rotary_dim;
    constexpr double kInvTwoPi = 0.15915494309189535;
    // the angle p * theta^(-2i/r), in turns, in fp64 (positions reach 10^5
    // and more, where an fp32 angle would already be off by ~10^-2 rad);
    // its fraction in [-1/2, 1/2] goes to the hardware sine and cosine,
    // which take turns.  The frequency is the product of the host's
    // theta^(-2 * 2^k / r) over the set bits k of i (at most seven fp64
    // products, ~1e-15 relative) instead of an fp64 exp2 and division per
    // element (0.6 us of the 256-sequence epilogue).
    auto angle = [&](int i, float& sn, float& c) __attribute__((always_inline)) {
      double freq = 1.0;
#pragma unroll
      for (int k = 0; k < 8; ++k) freq = (i >> k) & 1 ? freq * a.freq_pow2[k] : freq;
      const double turns = static_cast<double>(pos) * freq * kInvTwoPi;
      const float frac = static_cast<float>(turns - __builtin_rint(turns));
      sn = __builtin_amdgcn_sinf(frac);
      c = __builtin_amdgcn_cosf(frac);
    };
    if (E % 2 == 0 && !a.interleaved && r == D) {
      // rotation of the whole head in halves: the partner of element
      // lane + 64 j (j < E / 2) is lane + 64 (j + E / 2), in this lane, at
      // the same angle, so the pair turns in registers with one angle
      // (the same arithmetic as the exchange below)
#pragma unroll
      for (int j = 0; j < E / 2; ++j) {
        float sn, c;
        angle(lane + 64 * j, sn, c);
        const float x0 = v[j], x1 = v[j + E / 2];
        v[j] = x0 * c - x1 * sn;
        v[j + E / 2] = x1 * c + x0 * sn;
      }
    } else if (a.interleaved) {
      // interleaved pairs (e, e ^ 1): the partner is the neighbouring lane,
      // same register, fetched with a DPP swap of adjacent lanes (every
      // lane takes part, before the range test)
#pragma unroll
      for (int j = 0; j < E; ++j) {
        const float other = __builtin_bit_cast(
            float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v[j]), 0xB1, 0xF, 0xF, false));
        const int e = lane + 64 * j;
        if (e >= r) continue;
        float sn, c;
        angle(e >> 1, sn, c);
        v[j] = (e & 1) == 0 ? v[j] * c - other * sn : v[j] * c + other * sn;
      }
    } else {
#pragma unroll
      for (int j = 0; j < E; ++j) s[lane + 64 * j] = v[j];
      __syncthreads();
#pragma unroll
      for (int j = 0; j < E; ++j) {
        const int e = lane + 64 * j;
        if (e >= r) continue;
        // a partial rotation in halves: pairs (e, e + r / 2), across lanes
        const bool first = e < r / 2;
        const int i = first ? e : e - r / 2;
        const int partner = first ? e + r / 2 : e - r / 2;
        float sn, c;
        angle(i, sn, c);
        const float other = s[partner];
        v[j] = first ? v[j] * c - other * sn : v[j] * c + other * sn;
      }
    }
  }

  // outputs: q to q_out; k and v to k_out / v_out and, with a cache, to the page slot
  uint16_t* dst = nullptr;
  if (is_q) {
    dst = a.q_out + (static_cast<int64_t>(b) * a.hq + h) * D;
  } else {
    uint16_t* out = is_k ? a.k_out : a.v_out;
    if (out) dst = out + (static_cast<int64_t>(b) * a.hkv + g) * D;
  }
#pragma unroll
  for (int j = 0; j < E; ++j) {
    const uint16_t o = f32_to_bf16(v[j]);
    if (dst) dst[lane + 64 * j] = o;
    if (cache) cache[row + lane + 64 * j] = o;
  }
}

// Pass 1, one workgroup per (sequence b, chunk c of features), one feature
// per thread: z = y + residual (fp32 to scratch, bf16 to residual_out) and
// the chunk's sum of z^2 (fixed reduction order).  residual_out may be the
// residual buffer: each feature is read and written by the same thread.
template <int kSlots>
__global__ __launch_bounds__(kOProjChunk) void oproj_residual_kernel(OProjArgs a) {
  __shared__ float wsum[kOProjChunk / 64];
  const int chunks = oproj_chunks(a.hidden);
  const int b = blockIdx.x / chunks;
  const int c = blockIdx.x - b * chunks;
  const int n = c * kOProjChunk + threadIdx.x;
  const int64_t at = static_cast<int64_t>(b) * a.hidden + n;
  float z = 0.f;
  if (n < a.hidden) {
    const int rows[1] = {n};
    float y[1];
    gemv_rows<kSlots>(a.part, a.plan, a.batch, b, rows, y);
    z = y[0] + bf16_to_f32(a.residual[at]);
    a.z[at] = z;
    a.residual_out[at] = f32_to_bf16(z);
  }
  float ss = z * z;
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) ss += __shfl_xor(ss, off);
  if ((threadIdx.x & 63) == 0) wsum[threadIdx.x >> 6] = ss;
  __syncthreads();
  if (threadIdx.x == 0) {
    float t = 0.f;
#pragma unroll
    for (int i = 0; i < kOProjChunk / 64; ++i) t += wsum[i];
    a.chunk_ss[static_cast<int64_t>(b) * chunks + c] = t;
  }
}

// Pass 2, same grid: the sequence's total (chunk sums in chunk order) and
// h = z / sqrt(mean + eps) * w.
__global__ __launch_bounds__(kOProjChunk) void oproj_norm_kernel(OProjArgs a) {
  const int chunks = oproj_chunks(a.hidden);
  const int b = blockIdx.x / chunks;
  const int c = blockIdx.x - b * chunks;
  const int n = c * kOProjChunk + threadIdx.x;
  if (n >= a.hidden) return;
  // z and the weight are requested before the chunk sums (scalar loads,
  // eight in flight at a time), whose latency hides theirs
  const int64_t at = static_cast<int64_t>(b) * a.hidden + n;
  const float z = a.z[at];
  const float w = bf16_to_f32(a.norm_w[n]);
  const float* ss = a.chunk_ss + static_cast<int64_t>(b) * chunks;
  float tot = 0.f;
#pragma unroll 8
  for (int i = 0; i < chunks; ++i) tot += ss[i];
  const float inv = rsqrtf(tot / a.hidden + a.eps);
  a.normed_out[at] = f32_to_bf16(z * inv * w);
}

// The o_proj epilogue in one kernel for small batches, one workgroup per
// sequence b; thread t takes the four consecutive features 4 (t + 1024 j):
// z = y + residual kept in registers (fp32; bf16 to residual_out), the
// sequence's sum of z^2 reduced across the workgroup in a fixed order,
// then h = z / sqrt(mean + eps) * w.  Partials are read as 16-byte pieces.
template <int kSlots>
__global__ __launch_bounds__(kOProjOneThreads) void oproj_one_kernel(OProjArgs a) {
  constexpr int kGroups = kOProjOneFeatures / 4;  // groups of four features per thread, at most
  __shared__ float wsum[kOProjOneThreads / 64];
  const int b = blockIdx.x;
  const int tid = threadIdx.x;
  const int64_t base = static_cast<int64_t>(b) * a.hidden;
  float4 z[kGroups];
  uint2 w[kGroups];  // norm weights, requested with everything else before the reduction
  float ss = 0.f;
#pragma unroll
  for (int j = 0; j < kGroups; ++j) {
    const int n = 4 * (tid + kOProjOneThreads * j);
    z[j] = make_float4(0.f, 0.f, 0.f, 0.f);
    w[j] = make_uint2(0u, 0u);
    if (n < a.hidden) {
      w[j] = *reinterpret_cast<const uint2*>(a.norm_w + n);
      const uint2 r = *reinterpret_cast<const uint2*>(a.residual + base + n);
      const float4 y = gemv_rows4<kSlots>(a.part, a.plan, a.batch, b, n);
      z[j] = make_float4(y.x + bf16_to_f32(static_cast<uint16_t>(r.x)), y.y + bf16_to_f32(static_cast<uint16_t>(r.x >> 16)),
                         y.z + bf16_to_f32(static_cast<uint16_t>(r.y)), y.w + bf16_to_f32(static_cast<uint16_t>(r.y >> 16)));
      ss += z[j].x * z[j].x + z[j].y * z[j].y + z[j].z * z[j].z + z[j].w * z[j].w;
      uint2 o;
      o.x = f32_to_bf16(z[j].x) | (static_cast<uint32_t>(f32_to_bf16(z[j].y)) << 16);
      o.y = f32_to_bf16(z[j].z) | (static_cast<uint32_t>(f32_to_bf16(z[j].w)) << 16);
      *reinterpret_cast<uint2*>(a.residual_out + base + n) = o;
    }
  }
#pragma unroll
  for (int off = 32; off >= 1; off >>= 1) ss += __shfl_xor(ss, off);
  if ((tid & 63) == 0) wsum[tid >> 6] = ss;
  __syncthreads();
  float tot = 0.f;
#pragma unroll
  for (int i = 0; i < kOProjOneThreads / 64; ++i) tot += wsum[i];
  const float inv = rsqrtf(tot / a.hidden + a.eps);
#pragma unroll
  for (int j = 0; j < kGroups; ++j) {
    const int n = 4 * (tid + kOProjOneThreads * j);
    if (n < a.hidden) {
      uint2 o;
      o.x = f32_to_bf16(z[j].x * inv * bf16_to_f32(static_cast<uint16_t>(w[j].x))) |
            (static_cast<uint32_t>(f32_to_bf16(z[j].y * inv * bf16_to_f32(static_cast<uint16_t>(w[j].x >> 16)))) << 16);
      o.y = f32_to_bf16(z[j].z * inv * bf16_to_f32(static_cast<uint16_t>(w[j].y))) |
            (static_cast<uint32_t>(f32_to_bf16(z[j].w * inv * bf16_to_f32(static_cast<uint16_t>(w[j].y >> 16)))) << 16);
      *reinterpret_cast<uint2*>(a.normed_out + base + n) = o;
    }
  }
}


// The same for tile-major partials (the 256-sequence GEMV form), two
// sequences per workgroup: sequences 2i and 2i + 1 own the two 64-byte
// halves of every 128-byte line of their partials, so this workgroup reads
// whole lines that no other workgroup touches, where one workgroup per
// sequence fetched each line twice, on two CUs (256 x 5120: 10.6 against
// 14.4 us in kernel traces).  In each group of eight threads, thread q
// takes sequence 2i + q / 4 and features 4 (q % 4) .. +3 of a 16-feature
// piece.
template <int kSlots>
__global__ __launch_bounds__(kOProjOneThreads) void oproj_pair_kernel(OProjArgs a) {
  constexpr int kGroups = 2 * kOProjOneFeatures / 4;  // groups of four features per thread, at most
  constexpr int kPieces = kOProjOneThreads / 8;       // 16-feature pieces per round
  __shared__ float wsum[2][kOProjOneThreads / 64];
  const int tid = threadIdx.x;
  const int q = tid & 7;
  const int sq = q >> 2;
  const int b = 2 * blockIdx.x + sq;
  const bool live = b < a.batch;  // an odd batch: the last workgroup has one sequence
  const int64_t base = static_cast<int64_t>(b) * a.hidden;
  float4 z[kGroups];
  uint2 w[kGroups];
  float ss = 0.f;
#pragma unroll
  for (int j = 0; j < kGroups; ++j) {
    const int n = 16 * ((tid >> 3) + kPieces * j) + 4 * (q & 3);
    z[j] = make_float4(0.f, 0.f, 0.f, 0.f);
    w[j] = make_uint2(0u, 0u);
    if (live && n < a.hidden) {
      w[j] = *reinterpret_cast<const uint2*>(a.norm_w + n);
      const uint2 r = *reinterpret_cast<const uint2*>(a.residual + base + n);
      const float4 y = gemv_rows4<kSlots>(a.part, a.plan, a.batch, b, n);
      z[j] = make_float4(y.x + bf16_to_f32(static_cast<uint16_t>(r.x)), y.y + bf16_to_f32(static_cast<uint16_t>(r.x >> 16)),
                         y.z + bf16_to_f32(static_cast<uint16_t>(r.y)), y.w + bf16_to_f32(static_cast<uint16_t>(r.y >> 16)));
      ss += z[j].x * z[j].x + z[j].y * z[j].y + z[j].z * z[j].z + z[j].w * z[j].w;
      uint2 o;
      o.x = f32_to_bf16(z[j].x) | (static_cast<uint32_t>(f32_to_bf16(z[j].y)) << 16);
      o.y = f32_to_bf16(z[j].z) | (static_cast<uint32_t>(f32_to_bf16(z[j].w)) << 16);
      *reinterpret_cast<uint2*>(a.residual_out + base + n) = o;
    }
  }
  // per-sequence sums: the lanes of one sequence share bit 2 of the lane id
  ss += __shfl_xor(ss, 32);
  ss += __shfl_xor(ss, 16);
  ss += __shfl_xor(ss, 8);
  ss += __shfl_xor(ss, 2);
  ss += __shfl_xor(ss, 1);
  if ((tid & 63) == 0) wsum[0][tid >> 6] = ss;
  if ((tid & 63) == 4) wsum[1][tid >> 6] = ss;
  __syncthreads();
  float tot = 0.f;
#pragma unroll
  for (int i = 0; i < kOProjOneThreads / 64; ++i) tot += wsum[sq][i];
  const float inv = rsqrtf(tot / a.hidden + a.eps);
#pragma unroll
  for (int j = 0; j < kGroups; ++j) {
    const int n = 16 * ((tid >> 3) + kPieces * j) + 4 * (q & 3);
    if (live && n < a.hidden) {
      uint2 o;
      o.x = f32_to_bf16(z[j].x * inv * bf16_to_f32(static_cast<uint16_t>(w[j].x))) |
            (static_cast<uint32_t>(f32_to_bf16(z[j].y * inv * bf16_to_f32(static_cast<uint16_t>(w[j].x >> 16)))) << 16);
      o.y = f32_to_bf16(z[j].z * inv * bf16_to_f32(static_cast<uint16_t>(w[j].y))) |
            (static_cast<uint32_t>(f32_to_bf16(z[j].w * inv * bf16_to_f32(static_cast<uint16_t>(w[j].y >> 16)))) << 16);
      *reinterpret_cast<uint2*>(a.normed_out + base + n) = o;
    }
  }
}

}  // namespace

// Instantiations of the epilogues by the plan's partial slots per group.
template <int kSlots>
hipError_t launch_oproj_residual(const OProjArgs& a, hipStream_t st) {
  hipLaunchKernelGGL((oproj_residual_kernel<kSlots>), dim3(a.batch * oproj_chunks(a.hidden)), dim3(kOProjChunk), 0,
                     st, a);
  return hipGetLastError();
}

template <int D>
hipError_t launch_prelude(const PreludeArgs& a, hipStream_t st) {
  const dim3 grid(a.batch * (a.hq + 2 * a.hkv));
  if (a.plan.slots <= 4)
    hipLaunchKernelGGL((prelude_epilogue<D, 4>), grid, dim3(64), 0, st, a);
  else if (a.plan.slots <= 8)
    hipLaunchKernelGGL((prelude_epilogue<D, 8>), grid, dim3(64), 0, st, a);
  else if (a.plan.slots <= 12)
    hipLaunchKernelGGL((prelude_epilogue<D, 12>), grid, dim3(64), 0, st, a);
  else
    hipLaunchKernelGGL((prelude_epilogue<D, kGemvMaxSlots>), grid, dim3(64), 0, st, a);
  return hipGetLastError();
}

template <int kSlots>
hipError_t launch_oproj_one(const OProjArgs& a, hipStream_t st) {
  if (a.plan.seq_major)
    hipLaunchKernelGGL((oproj_one_kernel<kSlots>), dim3(a.batch), dim3(kOProjOneThreads), 0, st, a);
  else  // tile-major partials (the 256-sequence GEMV form): two sequences per workgroup
    hipLaunchKernelGGL((oproj_pair_kernel<kSlots>), dim3((a.batch + 1) / 2), dim3(kOProjOneThreads), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_oproj_epilogue(const OProjArgs& a, hipStream_t st) {
  // PDA_OPROJ_ONE=0 in the environment keeps the two passes at every batch (for measurement)
  static const bool one_ok = [] {
    const char* e = std::getenv("PDA_OPROJ_ONE");
    return !(e && e[0] == '0');
  }();
  // (the one-kernel form moves four bf16 features at a time: 8-byte aligned rows)
  const bool aligned8 = ((reinterpret_cast<uintptr_t>(a.residual) | reinterpret_cast<uintptr_t>(a.norm_w) |
                          reinterpret_cast<uintptr_t>(a.residual_out) | reinterpret_cast<uintptr_t>(a.normed_out)) &
                         7) == 0;
  if (one_ok && aligned8 && oproj_one_kernel(a.batch, a.hidden)) {
    return a.plan.slots <= 4   ? launch_oproj_one<4>(a, st)
           : a.plan.slots <= 8  ? launch_oproj_one<8>(a, st)
           : a.plan.slots <= 12 ? launch_oproj_one<12>(a, st)
                                : launch_oproj_one<kGemvMaxSlots>(a, st);
  }
  const dim3 grid(a.batch * oproj_chunks(a.hidden));
  const hipError_t e = a.plan.slots <= 4   ? launch_oproj_residual<4>(a, st)
                       : a.plan.slots <= 8  ? launch_oproj_residual<8>(a, st)
                       : a.plan.slots <= 12 ? launch_oproj_residual<12>(a, st)
                                            : launch_oproj_residual<kGemvMaxSlots>(a, st);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(oproj_norm_kernel, grid, dim3(kOProjChunk), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_pack(const uint16_t* w, uint16_t* wp, int n, int k, hipStream_t st) {
  const int64_t chunks = static_cast<int64_t>(n) * k / 8;
  const dim3 grid(static_cast<unsigned>((chunks + kPackThreads - 1) / kPackThreads));
  hipLaunchKernelGGL(pack_kernel, grid, dim3(kPackThreads), 0, st, w, wp, n, k);
  return hipGetLastError();
}

GemvPlan plan_gemv(int batch, int n, int k, int num_cus, bool seq_major) {
  GemvPlan p;
  const int nbt = (batch + 15) / 16;
  const int tiles = n / kTileRows;
  // Several row tiles per unit share each x fragment: as many as there are
  // 16-column batch tiles.  Within one batch tile of more than 4 sequences,
  // four, when every workgroup still gets at least kGemvGroupedUnits units
  // (x rows past the batch read as zeros with no traffic, so a few
  // sequences gain nothing; at 8 and 16 sequences four tiles per unit ran
  // 7% and 24% faster on 8192 x 8192 and 15% on 3072 x 5120, but 20% slower
  // on 3072 x 3072, where the larger partials of too few units per
  // workgroup cost more than the x reads saved).
  p.kt_count = k / kTileK;
  p.xlds = false;
  p.group = 1;
  // batches of more than 16: the thin-GEMM form when the row tiles split
  // into groups of kXWaves (PDA_GEMV_THIN=0 in the environment selects
  // gemv_kernel instead, for measurement, up to 64 sequences; above that
  // only the thin-GEMM form exists, and the callers check the rows)
  static const bool thin_ok = [] {
    const char* e = std::getenv("PDA_GEMV_THIN");
    return !(e && e[0] == '0');
  }();
  if ((thin_ok || nbt > 4) && nbt > 1 && tiles % kXWaves == 0) {
    p.xlds = true;
    p.group = kXWaves;
    p.units = static_cast<int64_t>(tiles / kXWaves) * p.kt_count;
    int64_t grid = static_cast<int64_t>(num_cus) * kXBlocksPerCu;
    const int64_t most = (p.units + kGemvMinTiles - 1) / kGemvMinTiles;  // >= kGemvMinTiles tiles per wave
    if (grid > most) grid = most;
    const int64_t cap = static_cast<int64_t>(kGemvMaxSlots - 1) * (tiles / kXWaves);
    if (grid > cap) grid = cap;
    if (grid < 1) grid = 1;
    p.grid = static_cast<int>(grid);
    p.blocks = grid;
    p.slots = static_cast<int>((static_cast<int64_t>(p.kt_count) * p.blocks + p.units - 1) / p.units + 1);
    // above 8 column tiles (gemv_thin_kernel) the partials stay tile-major:
    // sequence-major stores there made the 256-sequence GEMVs 15-20% slower
    p.seq_major = seq_major && nbt <= 8;
    return p;
  }
  if (nbt > 1 && tiles % nbt == 0) {
    p.group = nbt;
  } else if (nbt == 1 && batch > 4 && tiles % 4 == 0 &&
             static_cast<int64_t>(tiles / 4) * p.kt_count >=
                 static_cast<int64_t>(kGemvGroupedUnits) * num_cus * gemv_blocks_per_cu(1, 4)) {
    p.group = 4;
  }
  p.units = static_cast<int64_t>(tiles / p.group) * p.kt_count;
  // workgroups resident per CU: the kernel's registers (its launch bounds)
  // and the LDS of the cross-wave reduction (4 waves x group x column tiles
  // x 1 KB) both limit it; a grid larger than what is resident would run in
  // two rounds
  const int lds = kGemvWaves * p.group * nbt * 1024;
  int per_cu = (160 * 1024) / lds;
  const int regs = gemv_blocks_per_cu(nbt, p.group);
  per_cu = per_cu < regs ? per_cu : regs;
  int64_t grid = static_cast<int64_t>(num_cus) * per_cu;
  const int64_t most = (p.units + static_cast<int64_t>(kGemvWaves) * kGemvMinTiles - 1) /
                       (static_cast<int64_t>(kGemvWaves) * kGemvMinTiles);
  if (grid > most) grid = most;
  // at most kGemvMaxSlots workgroups per row group: blocks <= (kGemvMaxSlots - 1) * groups
  const int64_t cap = static_cast<int64_t>(kGemvMaxSlots - 1) * (tiles / p.group);
  if (grid > cap) grid = cap;
  if (grid < 1) grid = 1;
  p.grid = static_cast<int>(grid);
  p.blocks = grid;
  // workgroups touching one row group: its kt_count units span at most this many ranges
  p.slots = static_cast<int>((static_cast<int64_t>(p.kt_count) * p.blocks + p.units - 1) / p.units + 1);
  p.seq_major = seq_major;
  return p;
}

int64_t gemv_partial_floats(const GemvPlan& p, int batch, int n) {
  return static_cast<int64_t>(n / kTileRows) * p.slots * batch * kTileRows;  // groups * group tiles = n / 16
}

template <int kNBT>
hipError_t launch_xlds(const GemvArgs& a, hipStream_t st) {
  constexpr int lds = gemv_xlds_lds_bytes(kNBT);
  // the dynamic-LDS limit is raised once per device (bit = device ordinal)
  static std::atomic<uint64_t> attr_set{0};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  const uint64_t bit = dev < 64 ? uint64_t{1} << dev : 0;
  if (!bit || !(attr_set.load() & bit)) {
    e = hipFuncSetAttribute(reinterpret_cast<const void*>(&gemv_xlds_kernel<kNBT>),
                            hipFuncAttributeMaxDynamicSharedMemorySize, lds);
    if (e != hipSuccess) return e;
    attr_set.fetch_or(bit);
  }
  hipLaunchKernelGGL((gemv_xlds_kernel<kNBT>), dim3(a.plan.grid), dim3(kXWaves * 64), lds, st, a.x, a.wp, a.part,
                     a.batch, a.n, a.k, a.plan.slots, a.plan.seq_major ? 1 : 0);
  return hipGetLastError();
}

template <int kNBT, int kW, int kR, int kC, int kD>
hipError_t launch_thin(const GemvArgs& a, hipStream_t st) {
  constexpr int lds = (kD + 1) * kC * kNBT * 1024;
  static std::atomic<uint64_t> attr_set{0};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  const uint64_t bit = dev < 64 ? uint64_t{1} << dev : 0;
  if (!bit || !(attr_set.load() & bit)) {
    e = hipFuncSetAttribute(reinterpret_cast<const void*>(&gemv_thin_kernel<kNBT, kW, kR, kC, kD>),
                            hipFuncAttributeMaxDynamicSharedMemorySize, lds);
    if (e != hipSuccess) return e;
    attr_set.fetch_or(bit);
  }
  hipLaunchKernelGGL((gemv_thin_kernel<kNBT, kW, kR, kC, kD>), dim3(a.plan.grid), dim3(kW * 64), lds, st, a.x, a.wp,
                     a.part, a.batch, a.n, a.k, a.plan.slots);
  return hipGetLastError();
}

hipError_t launch_gemv(const GemvArgs& a, hipStream_t st) {
  const dim3 grid(a.plan.grid);
  const int nbt = (a.batch + 15) / 16;
  const int sl = a.plan.slots;
  // Above 128 sequences the LDS-copy form with two row tiles per wave: on
  // the 256-sequence prelude (5120 -> 7168) it ran 40.8 against 46.2 us for
  // gemv_xlds_kernel<16>, on the o_proj (5120 -> 5120) 31.4 against 33.0.
  // Up to 128 sequences gemv_xlds_kernel is the faster form (batch 64,
  // 4096 -> 6144: 15.1 us against 17.1 for the LDS-copy form at its best
  // depth).
  if (a.plan.xlds) {
    if (nbt == 2) return launch_xlds<2>(a, st);
    if (nbt == 3) return launch_xlds<3>(a, st);
    if (nbt == 4) return launch_xlds<4>(a, st);
    if (nbt <= 8) return launch_xlds<8>(a, st);  // column tiles past the batch read zeros
    return launch_thin<16, 4, 2, 1, 4>(a, st);
  }
  if (nbt > 4) return hipErrorInvalidValue;  // above 64 sequences only the thin-GEMM form
  const bool grouped = a.plan.group > 1;
#define PDA_GEMV(NBT, R) \
  hipLaunchKernelGGL((gemv_kernel<NBT, R>), grid, dim3(kGemvThreads), 0, st, a.x, a.wp, a.part, a.batch, a.n, a.k, sl, \
                     a.plan.seq_major ? 1 : 0)
  switch (nbt) {
    case 1: if (grouped) PDA_GEMV(1, 4); else PDA_GEMV(1, 1); break;
    case 2: if (grouped) PDA_GEMV(2, 2); else PDA_GEMV(2, 1); break;
    case 3: if (grouped) PDA_GEMV(3, 3); else PDA_GEMV(3, 1); break;
    default: if (grouped) PDA_GEMV(4, 4); else PDA_GEMV(4, 1); break;
  }
#undef PDA_GEMV
  return hipGetLastError();
}

hipError_t launch_prelude_epilogue(const PreludeArgs& a, hipStream_t st) {
  if (a.d == 64) return launch_prelude<64>(a, st);
  if (a.d == 128) return launch_prelude<128>(a, st);
  return launch_prelude<256>(a, st);
}

}  // namespace pda
