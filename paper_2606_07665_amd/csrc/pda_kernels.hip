// Paged decode attention kernels for MI355X (gfx950, CDNA4, wave64).
//
// What is computed: the paper's kernel family (iv), decode attention over a
// paged KV cache with grouped-query heads (Method, "Principle-Driven LLM
// Kernel Generator"): per sequence and kv head, an online softmax over the
// cached tokens, split across many workers and merged by log-sum-exp
// ("cross-CTA merging").  The CUDA design the paper sketches (appendix:
// m16n8k16 fragments, ldmatrix, padded shared rows, a fence-based merge) is
// prior art for another GPU; this file is laid out for CDNA4 instead:
//
//  * Work split (stream-K over the context).  The flattened space of
//    (sequence b, kv head g, 32-token step) is cut into equal contiguous
//    ranges, one per wave.  Every wave gets the same number of steps (+-1)
//    whatever the length mix, so ragged batches stay balanced, and a wave
//    that covers a whole (b, g) writes the final output itself.  A wave that
//    covers part of one writes a partial (running max, sum, unnormalised
//    accumulator) to a slot indexed wave + sequence, which is unique because
//    each wave's range is contiguous.
//  * QK^T on the matrix cores: v_mfma_f32_16x16x32_bf16 with the 16 keys of
//    a tile as the A rows (each lane loads 16 contiguous bytes of one key
//    row straight from HBM, exactly the A-operand layout) and the query
//    heads of the GQA group as the B columns (zero-padded to 16).  One K
//    read serves every head of the group.
//  * The softmax runs in the MFMA result layout (lane = head column, four
//    key rows per lane), which is lane-for-lane the B-operand layout the
//    P.V product needs, so probabilities never move between lanes.
//  * V is staged through LDS (padded rows) and read back transposed with
//    ds_read_b64_tr_b16 to form the A operand of O^T = V^T P^T, again on
//    v_mfma_f32_16x16x32_bf16.  The output accumulator lands with the head
//    in the lane column, so the online-softmax rescale is a per-lane scalar.
//  * Merge: a second small kernel combines the partials of each (b, g) with
//    exp2 weights.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "pda_internal.h"

namespace pda {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef short i16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned u32x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;

constexpr float kLog2e = 1.4426950408889634f;

template <int D>
struct Shape {
  static constexpr int kQK = D / 32;            // MFMAs per 16-key tile for QK^T
  static constexpr int kDT = D / 16;            // 16-wide d tiles of the output
  static constexpr int kChunks = D / 8;         // 16-byte chunks per key/value row
  static constexpr int kRowsPerLoad = 64 / kChunks;      // V rows per wave load
  static constexpr int kVLoads = kStep / kRowsPerLoad;   // V loads per step
  static constexpr int kRowBytes = 2 * D + 32;  // padded LDS row of the V tile
  static constexpr int kTileBytes = kStep * kRowBytes;
};

__device__ __forceinline__ int uniform(int x) { return __builtin_amdgcn_readfirstlane(x); }

__device__ __forceinline__ int clamp_len(int L, int max_ctx) {
  return L < 0 ? 0 : (L > max_ctx ? max_ctx : L);
}

__device__ __forceinline__ u32x4 ld16(const uint16_t* p) {
  return *reinterpret_cast<const u32x4*>(p);
}

// physical page of logical page j of a sequence, clamped so that a bad page
// table entry or a token past the end can never address outside the pool
__device__ __forceinline__ int page_at(const int32_t* __restrict__ bt_row, int j, int npages,
                                      int num_pages) {
  j = j < npages ? j : npages - 1;
  unsigned p = static_cast<unsigned>(bt_row[j]);
  return static_cast<int>(p < static_cast<unsigned>(num_pages) ? p : num_pages - 1);
}

template <int D, bool kLanePages>
__global__ __launch_bounds__(kBlockThreads, 2) void split_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ kc,
    const uint16_t* __restrict__ vc, const int32_t* __restrict__ bt,
    const int32_t* __restrict__ lens, uint16_t* __restrict__ out,
    float* __restrict__ ws_acc, float* __restrict__ ws_ml, int32_t* __restrict__ ws_pref,
    int batch, int hq, int hkv, int group, int page_shift, int num_pages, int maxp,
    int min_steps, float scale_log2) {
  using S = Shape<D>;
  extern __shared__ __align__(16) unsigned char smem[];
  int32_t* pref = reinterpret_cast<int32_t*>(smem + kWavesPerBlock * S::kTileBytes);
  int32_t* scan = reinterpret_cast<int32_t*>(smem);  // reuses the V tiles before the loop

  const int tid = threadIdx.x;
  const int page = 1 << page_shift;
  const int max_ctx = maxp << page_shift;

  // ---- per-block prefix over the batch of 32-token steps per sequence ----
  {
    const int per = (batch + kBlockThreads - 1) / kBlockThreads;
    const int lo = tid * per;
    const int hi = min(batch, lo + per);
    int sum = 0;
    for (int b = lo; b < hi; ++b) sum += (clamp_len(lens[b], max_ctx) + kStep - 1) / kStep;
    scan[tid] = sum;
    __syncthreads();
    for (int off = 1; off < kBlockThreads; off <<= 1) {
      int v = tid >= off ? scan[tid - off] : 0;
      __syncthreads();
      scan[tid] += v;
      __syncthreads();
    }
    int run = scan[tid] - sum;
    for (int b = lo; b < hi; ++b) {
      pref[b] = run;
      run += (clamp_len(lens[b], max_ctx) + kStep - 1) / kStep;
    }
    if (tid == kBlockThreads - 1) pref[batch] = scan[tid];
    __syncthreads();
    if (blockIdx.x == 0)
      for (int b = tid; b <= batch; b += kBlockThreads) ws_pref[b] = pref[b];
    __syncthreads();  // the scan area is overwritten by V tiles below
  }

  const int lane = tid & 63;
  const int wid = tid >> 6;
  const int g4 = lane >> 4;  // lane group: MFMA k block / C row block
  const int c = lane & 15;   // MFMA row (A) / column (B, C)

  const int64_t total = static_cast<int64_t>(uniform(pref[batch])) * hkv;
  if (total == 0) return;
  const int64_t nwaves = static_cast<int64_t>(gridDim.x) * kWavesPerBlock;
  int64_t weff = (total + min_steps - 1) / min_steps;
  weff = weff < nwaves ? weff : nwaves;
  const int w = blockIdx.x * kWavesPerBlock + wid;
  if (w >= weff) return;
  int64_t x = (static_cast<int64_t>(w) * total) / weff;
  const int64_t xend = (static_cast<int64_t>(w + 1) * total) / weff;

  // sequence containing step x: largest b with pref[b] * hkv <= x
  int b;
  {
    const int y = static_cast<int>(x / hkv);
    int lo = 0, hi = batch - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (uniform(pref[mid]) <= y) lo = mid; else hi = mid - 1;
    }
    b = lo;
  }
  int nb = uniform(pref[b + 1]) - uniform(pref[b]);
  int rel = static_cast<int>(x - static_cast<int64_t>(uniform(pref[b])) * hkv);
  int g = rel / nb;
  int s0 = rel - g * nb;

  unsigned char* vtile = smem + wid * S::kTileBytes;
  const int vr = lane / S::kChunks;   // V row within one wave load
  const int vq = lane % S::kChunks;   // 16-byte chunk within the row
  const int64_t tok_stride = static_cast<int64_t>(hkv) * D;       // elements per token
  const int64_t page_stride = tok_stride << page_shift;            // elements per page

  while (true) {
    const int64_t remaining = xend - x;
    const int s1 = remaining < nb - s0 ? s0 + static_cast<int>(remaining) : nb;
    const int L = uniform(clamp_len(lens[b], max_ctx));
    const int npages = (L + page - 1) >> page_shift;
    const int32_t* bt_row = bt + static_cast<int64_t>(b) * maxp;

    // query operand (B of QK^T): head c of the group, d = 32*kk + 8*g4 + e
    bf16x8 qop[S::kQK];
    {
      const uint16_t* qrow = q + (static_cast<int64_t>(b) * hq + g * group + c) * D + 8 * g4;
#pragma unroll
      for (int kk = 0; kk < S::kQK; ++kk) {
        u32x4 v = {0u, 0u, 0u, 0u};
        if (c < group) v = ld16(qrow + 32 * kk);
        qop[kk] = __builtin_bit_cast(bf16x8, v);
      }
    }
    const uint16_t* kg = kc + static_cast<int64_t>(g) * D;
    const uint16_t* vg = vc + static_cast<int64_t>(g) * D;

    f32x4 acc[S::kDT];
#pragma unroll
    for (int dt = 0; dt < S::kDT; ++dt) acc[dt] = f32x4{0.f, 0.f, 0.f, 0.f};
    float m_run = -__builtin_inff();
    float l_lane = 0.f;

    for (int s = s0; s < s1; ++s) {
      const int t0 = s * kStep;
      // ---------------- loads: 2 K tiles in A layout, V rows for LDS
      u32x4 kreg[2][S::kQK];
      u32x4 vreg[S::kVLoads];
      if constexpr (!kLanePages) {
        // pages of 16 or more tokens: each 16-token half of the step lies in one page
        const int pA = uniform(page_at(bt_row, t0 >> page_shift, npages, num_pages));
        const int pB = uniform(page_at(bt_row, (t0 + 16) >> page_shift, npages, num_pages));
#pragma unroll
        for (int T = 0; T < 2; ++T) {
          const int tok = t0 + 16 * T + c;
          const int64_t off = (T ? pB : pA) * page_stride + (tok & (page - 1)) * tok_stride + 8 * g4;
#pragma unroll
          for (int kk = 0; kk < S::kQK; ++kk) kreg[T][kk] = ld16(kg + off + 32 * kk);
        }
#pragma unroll
        for (int i = 0; i < S::kVLoads; ++i) {
          const int tau = S::kRowsPerLoad * i + vr;
          const int tok = t0 + tau;
          const int64_t off = ((tau >> 4) ? pB : pA) * page_stride + (tok & (page - 1)) * tok_stride + 8 * vq;
          vreg[i] = ld16(vg + off);
        }
      } else {
        // small pages: every lane looks up the page of its own token
#pragma unroll
        for (int T = 0; T < 2; ++T) {
          const int tok = t0 + 16 * T + c;
          const int pg = page_at(bt_row, tok >> page_shift, npages, num_pages);
          const int64_t off = pg * page_stride + (tok & (page - 1)) * tok_stride + 8 * g4;
#pragma unroll
          for (int kk = 0; kk < S::kQK; ++kk) kreg[T][kk] = ld16(kg + off + 32 * kk);
        }
#pragma unroll
        for (int i = 0; i < S::kVLoads; ++i) {
          const int tok = t0 + S::kRowsPerLoad * i + vr;
          const int pg = page_at(bt_row, tok >> page_shift, npages, num_pages);
          const int64_t off = pg * page_stride + (tok & (page - 1)) * tok_stride + 8 * vq;
          vreg[i] = ld16(vg + off);
        }
      }
      const bool tail = t0 + kStep > L;

      // ---------------- V rows -> LDS (rows past the end are zeroed, never NaN*0)
#pragma unroll
      for (int i = 0; i < S::kVLoads; ++i) {
        const int tau = S::kRowsPerLoad * i + vr;
        u32x4 v = vreg[i];
        if (tail && t0 + tau >= L) v = u32x4{0u, 0u, 0u, 0u};
        *reinterpret_cast<u32x4*>(vtile + tau * S::kRowBytes + 16 * vq) = v;
      }

      // ---------------- S^T = K Q^T : rows = keys 16T + 4*g4 + i, column = head c
      f32x4 sacc[2];
#pragma unroll
      for (int T = 0; T < 2; ++T) {
        sacc[T] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kk = 0; kk < S::kQK; ++kk)
          sacc[T] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
              __builtin_bit_cast(bf16x8, kreg[T][kk]), qop[kk], sacc[T], 0, 0, 0);
      }

      // ---------------- online softmax in log2 units
      float sv[2][4];
      float mx = -__builtin_inff();
#pragma unroll
      for (int T = 0; T < 2; ++T)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          float v = sacc[T][i] * scale_log2;
          if (tail && t0 + 16 * T + 4 * g4 + i >= L) v = -__builtin_inff();
          sv[T][i] = v;
          mx = fmaxf(mx, v);
        }
      mx = fmaxf(mx, __shfl_xor(mx, 16));
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      const float m_new = fmaxf(m_run, mx);
      const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
      m_run = m_new;
      bf16x8 pop;
      float psum = 0.f;
#pragma unroll
      for (int T = 0; T < 2; ++T)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const __bf16 pb = static_cast<__bf16>(__builtin_amdgcn_exp2f(sv[T][i] - m_new));
          pop[4 * T + i] = pb;
          psum += static_cast<float>(pb);
        }
      l_lane = l_lane * alpha + psum;
#pragma unroll
      for (int dt = 0; dt < S::kDT; ++dt) acc[dt] *= alpha;

      // ---------------- O^T += V^T P^T ; V^T operand via transposed LDS reads
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
      {
        const unsigned char* r0 = vtile + (4 * g4 + (c >> 2)) * S::kRowBytes + 8 * (c & 3);
        const unsigned char* r1 = r0 + 16 * S::kRowBytes;
#pragma unroll
        for (int dt = 0; dt < S::kDT; ++dt) {
          const i16x4 a0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(r0 + 32 * dt));
          const i16x4 a1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(r1 + 32 * dt));
          const i16x8 a = __builtin_shufflevector(a0, a1, 0, 1, 2, 3, 4, 5, 6, 7);
          acc[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), pop,
                                                             acc[dt], 0, 0, 0);
        }
      }
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    }

    // ---------------- epilogue for this (b, g) piece
    float l_tot = l_lane + __shfl_xor(l_lane, 16);
    l_tot += __shfl_xor(l_tot, 32);
    const bool whole = (s0 == 0) && (s1 == nb);
    if (c < group) {
      const int h = g * group + c;
      if (whole) {
        const float inv = 1.0f / l_tot;
        uint16_t* orow = out + (static_cast<int64_t>(b) * hq + h) * D + 4 * g4;
#pragma unroll
        for (int dt = 0; dt < S::kDT; ++dt) {
          typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
          bf16x4 o;
#pragma unroll
          for (int i = 0; i < 4; ++i) o[i] = static_cast<__bf16>(acc[dt][i] * inv);
          *reinterpret_cast<u32x2*>(orow + 16 * dt) = __builtin_bit_cast(u32x2, o);
        }
      } else {
        const int64_t slot = static_cast<int64_t>(w) + static_cast<int64_t>(b) * hkv + g;
        float* arow = ws_acc + (slot * group + c) * D + 4 * g4;
#pragma unroll
        for (int dt = 0; dt < S::kDT; ++dt) *reinterpret_cast<f32x4*>(arow + 16 * dt) = acc[dt];
        if (g4 == 0) {
          ws_ml[(slot * group + c) * 2 + 0] = m_run;
          ws_ml[(slot * group + c) * 2 + 1] = l_tot;
        }
      }
    }

    x += s1 - s0;
    if (x >= xend) break;
    s0 = 0;
    if (++g == hkv) {
      g = 0;
      do {
        ++b;
        nb = uniform(pref[b + 1]) - uniform(pref[b]);
      } while (nb == 0);
    }
  }
}

// Combine the partials of one (b, g): out = sum_j 2^(m_j - M) acc_j / sum_j 2^(m_j - M) l_j.
// Also writes the zero rows of empty sequences.
template <int D>
__global__ __launch_bounds__(kBlockThreads) void merge_kernel(
    uint16_t* __restrict__ out, const float* __restrict__ ws_acc, const float* __restrict__ ws_ml,
    const int32_t* __restrict__ ws_pref, int batch, int hq, int hkv, int group, int min_steps,
    int split_waves) {
  const int s = blockIdx.x;
  const int b = s / hkv;
  const int g = s - b * hkv;
  const int nb = ws_pref[b + 1] - ws_pref[b];
  const int tid = threadIdx.x;
  constexpr int kQuads = D / 4;
  constexpr int kHeadsPerPass = kBlockThreads / kQuads;
  const int hh0 = tid / kQuads;
  const int d4 = (tid % kQuads) * 4;
  typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));

  if (nb == 0) {
    for (int hh = hh0; hh < group; hh += kHeadsPerPass) {
      uint16_t* orow = out + (static_cast<int64_t>(b) * hq + g * group + hh) * D + d4;
      *reinterpret_cast<u32x2*>(orow) = u32x2{0u, 0u};
    }
    return;
  }
  const int64_t total = static_cast<int64_t>(ws_pref[batch]) * hkv;
  int64_t weff = (total + min_steps - 1) / min_steps;
  weff = weff < split_waves ? weff : split_waves;
  const int64_t x0 = static_cast<int64_t>(ws_pref[b]) * hkv + static_cast<int64_t>(g) * nb;
  const int64_t x1 = x0 + nb - 1;
  const int64_t w0 = ((x0 + 1) * weff - 1) / total;
  const int64_t w1 = ((x1 + 1) * weff - 1) / total;
  if (w0 == w1) return;  // one wave covered the sequence and wrote it

  for (int hh = hh0; hh < group; hh += kHeadsPerPass) {
    float big_m = -__builtin_inff();
    for (int64_t w = w0; w <= w1; ++w)
      big_m = fmaxf(big_m, ws_ml[((w + s) * group + hh) * 2]);
    float den = 0.f;
    f32x4 num = {0.f, 0.f, 0.f, 0.f};
    for (int64_t w = w0; w <= w1; ++w) {
      const int64_t slot = w + s;
      const float f = __builtin_amdgcn_exp2f(ws_ml[(slot * group + hh) * 2] - big_m);
      den += f * ws_ml[(slot * group + hh) * 2 + 1];
      num += f * *reinterpret_cast<const f32x4*>(ws_acc + (slot * group + hh) * D + d4);
    }
    const float inv = 1.0f / den;
    bf16x4 o;
#pragma unroll
    for (int i = 0; i < 4; ++i) o[i] = static_cast<__bf16>(num[i] * inv);
    uint16_t* orow = out + (static_cast<int64_t>(b) * hq + g * group + hh) * D + d4;
    *reinterpret_cast<u32x2*>(orow) = __builtin_bit_cast(u32x2, o);
  }
}

template <int D, bool kLanePages>
static hipError_t launch_split(const LaunchArgs& a, hipStream_t st) {
  using S = Shape<D>;
  const size_t lds = static_cast<size_t>(kWavesPerBlock) * S::kTileBytes +
                     static_cast<size_t>(a.batch + 1) * sizeof(int32_t);
  static bool attr_set = false;
  if (!attr_set) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&split_kernel<D, kLanePages>),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, kMaxLdsBytes);
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  hipLaunchKernelGGL((split_kernel<D, kLanePages>), dim3(a.grid), dim3(kBlockThreads), lds, st,
                     a.q, a.k, a.v, a.bt, a.lens, a.out, a.ws_acc, a.ws_ml, a.ws_pref, a.batch,
                     a.hq, a.hkv, a.group, a.page_shift, a.num_pages, a.maxp, a.min_steps,
                     a.scale * kLog2e);
  return hipGetLastError();
}

template <int D>
static hipError_t launch_merge(const LaunchArgs& a, hipStream_t st) {
  hipLaunchKernelGGL((merge_kernel<D>), dim3(a.batch * a.hkv), dim3(kBlockThreads), 0, st, a.out,
                     a.ws_acc, a.ws_ml, a.ws_pref, a.batch, a.hq, a.hkv, a.group, a.min_steps,
                     a.grid * kWavesPerBlock);
  return hipGetLastError();
}

hipError_t launch_split_kernel(const LaunchArgs& a, hipStream_t st) {
  const bool lane_pages = a.page_shift < 4;
  if (a.head_dim == 128) return lane_pages ? launch_split<128, true>(a, st) : launch_split<128, false>(a, st);
  return lane_pages ? launch_split<64, true>(a, st) : launch_split<64, false>(a, st);
}

hipError_t launch_merge_kernel(const LaunchArgs& a, hipStream_t st) {
  if (a.head_dim == 128) return launch_merge<128>(a, st);
  return launch_merge<64>(a, st);
}

size_t split_lds_bytes(int head_dim, int batch) {
  const size_t tile = head_dim == 128 ? Shape<128>::kTileBytes : Shape<64>::kTileBytes;
  return kWavesPerBlock * tile + static_cast<size_t>(batch + 1) * sizeof(int32_t);
}

}  // namespace pda
