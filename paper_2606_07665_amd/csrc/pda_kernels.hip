// Paged decode attention kernel for MI355X (gfx950, CDNA4, wave64).
//
// What is computed: the paper's kernel family (iv), decode attention over a
// paged KV cache with grouped-query heads (Method, "Principle-Driven LLM
// Kernel Generator"): per sequence and kv head, an online softmax over the
// cached tokens, split across many workers, then a log-sum-exp merge of the
// splits done inside the same kernel ("fused cross-CTA merging"; the paper's
// appendix describes a fence-based merge with no separate reduction kernel).
// The CUDA design the paper sketches (m16n8k16 fragments, ldmatrix, padded
// shared rows) is prior art for another GPU; this kernel is laid out for
// CDNA4 instead:
//
//  * Work split (stream-K over the context).  The flattened space of
//    (sequence b, kv head g, 32-token step) is cut into equal contiguous
//    ranges, one per workgroup of four wave64 workers, so every workgroup
//    gets the same amount of KV whatever the length mix.  Inside a range the
//    four waves take interleaved steps, each running its own online softmax.
//  * QK^T on the matrix cores: v_mfma_f32_16x16x32_bf16 with the 16 keys of
//    a tile as A rows (each lane loads 16 contiguous bytes of one key row
//    straight from HBM, which is the A-operand layout) and the query heads
//    of the GQA group as B columns (zero-padded to 16).  One K read serves
//    every head of the group.
//  * The softmax runs in the MFMA result layout (lane = head column, four
//    key rows per lane), which is lane-for-lane the B operand of the P.V
//    product, so probabilities never move between lanes.
//  * V is staged through LDS (padded rows) and read back transposed with
//    ds_read_b64_tr_b16 to form the A operand of O^T = V^T P^T.  The output
//    accumulator has the head in the lane column, so the online-softmax
//    rescale is one scalar per lane.
//  * Software pipeline: the K/V loads of a wave's next step are issued
//    before its current step is computed, and the page ids two steps ahead
//    before that, so the loop body is one basic block whose waits are all
//    satisfied by issue order.
//  * Merge: at the end of a (b, g) piece the four waves combine in LDS.  If
//    the workgroup covered the whole sequence it writes the output; else it
//    writes one partial (max in log2 units, sum, unnormalised accumulator)
//    to a slot indexed workgroup + sequence (unique because ranges are
//    contiguous) with write-through agent-scope stores, waits for them to be
//    acknowledged and bumps a per-sequence counter.  The workgroup that
//    brings the counter to the number of pieces merges all pieces in slot
//    order (so the result does not depend on arrival order), reading them
//    from the agent coherence point, and resets the counter.  No L2-wide
//    writeback or invalidate is issued (those cost more than the merge).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "pda_internal.h"

namespace pda {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef short i16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
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
  // Padded LDS rows.  K rows (stride 2D+16 bytes): the A-operand read of a
  // 16-row tile (lane = row, 16 B each) then starts every row 4 banks apart.
  // V rows (stride 2D+32 bytes): the transposed reads of 8 rows x 32 B start
  // every row 8 banks apart.
  static constexpr int kKRowBytes = 2 * D + 16;
  static constexpr int kVRowBytes = 2 * D + 32;
  static constexpr int kKTileBytes = kStep * kKRowBytes;
  static constexpr int kVTileBytes = kStep * kVRowBytes;
  static constexpr int kTileBytes = kKTileBytes + kVTileBytes;   // per wave
  static constexpr int kAccBytes = 64 * kDT * 16;        // one wave's accumulator in LDS
  static_assert(kAccBytes <= kTileBytes, "accumulator exchange reuses the K/V tiles");
  // LDS layout: [4 x (K tile, V tile)][ml exchange 4 x 16 x 2 floats][flag][prefix]
  static constexpr int kMlOff = kWavesPerBlock * kTileBytes;
  static constexpr int kFlagOff = kMlOff + kWavesPerBlock * 16 * 2 * 4;
  static constexpr int kPrefOff = kFlagOff + 16;
};

__device__ __forceinline__ int uniform(int x) { return __builtin_amdgcn_readfirstlane(x); }

__device__ __forceinline__ int clamp_len(int L, int max_ctx) {
  return L < 0 ? 0 : (L > max_ctx ? max_ctx : L);
}

__device__ __forceinline__ u32x4 ld16(const uint16_t* p) {
  return *reinterpret_cast<const u32x4*>(p);
}

// K and V are read exactly once per call, with raw buffer loads:
//  * non-temporal (cache policy NT): on MI355X a plain streaming read runs at
//    ~7.1 TB/s this way against ~6.1 TB/s with default loads;
//  * the descriptor's base is the page (a wave-uniform 64-bit address) and
//    its size covers only the valid token rows, so rows past the end of the
//    sequence, or a whole step that does not exist, read as zeros without
//    touching memory.
constexpr int kBufferDword3 = 0x00020000;  // raw buffer, 32-bit data format (gfx9 family)
constexpr int kCachePolicyNT = 2;

__device__ __forceinline__ __amdgpu_buffer_rsrc_t page_rsrc(const uint16_t* base, int bytes) {
  // the base is wave-uniform; passing it through readfirstlane keeps the
  // descriptor in SGPRs (a 64-bit VALU add would otherwise leave it in VGPRs
  // and every load would be wrapped in a waterfall loop)
  const uint64_t a = reinterpret_cast<uint64_t>(base);
  const uint32_t lo = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(a));
  const uint32_t hi = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(a >> 32));
  void* ub = reinterpret_cast<void*>((static_cast<uint64_t>(hi) << 32) | lo);
  return __builtin_amdgcn_make_buffer_rsrc(ub, 0, uniform(bytes), kBufferDword3);
}
__device__ __forceinline__ u32x4 ld16_stream(__amdgpu_buffer_rsrc_t r, int byte_off) {
  return __builtin_amdgcn_raw_buffer_load_b128(r, byte_off, 0, kCachePolicyNT);
}

// Split partials cross workgroups that may sit on different XCDs, whose L2
// caches are not coherent with each other.  They are written and read only
// with agent-scope relaxed atomic accesses (write-through stores and loads
// from the agent coherence point, sc1 on gfx950), so no L2 writeback or
// invalidate of the whole cache is needed around the arrival counter.
__device__ __forceinline__ void store_agent(float* p, float v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float load_agent(const float* p) {
  return __hip_atomic_load(const_cast<float*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
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
    float* __restrict__ ws_acc, float* __restrict__ ws_ml, int32_t* __restrict__ ws_cnt,
    int batch, int hq, int hkv, int group, int page_shift, int num_pages, int maxp,
    int min_steps, float scale_log2) {
  using S = Shape<D>;
  extern __shared__ __align__(16) unsigned char smem[];
  int32_t* pref = reinterpret_cast<int32_t*>(smem + S::kPrefOff);
  float* ml_x = reinterpret_cast<float*>(smem + S::kMlOff);
  int32_t* flag = reinterpret_cast<int32_t*>(smem + S::kFlagOff);
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
  }
  // empty sequences have no steps: block 0 writes their zero rows
  if (blockIdx.x == 0) {
    const int row16 = hq * D / 8;  // 16-byte stores per sequence
    for (int b = 0; b < batch; ++b) {
      if (pref[b + 1] != pref[b]) continue;
      u32x4* orow = reinterpret_cast<u32x4*>(out + static_cast<int64_t>(b) * hq * D);
      for (int i = tid; i < row16; i += kBlockThreads) orow[i] = u32x4{0u, 0u, 0u, 0u};
    }
  }

  const int lane = tid & 63;
  const int wid = uniform(tid >> 6);  // wave-uniform: lets the compiler keep per-wave values in SGPRs
  const int g4 = lane >> 4;  // lane group: MFMA k block / C row block
  const int c = lane & 15;   // MFMA row (A) / column (B, C)

  const int64_t total = static_cast<int64_t>(pref[batch]) * hkv;
  if (total == 0) return;
  const int64_t per_block_min = static_cast<int64_t>(min_steps) * kWavesPerBlock;
  int64_t beff = (total + per_block_min - 1) / per_block_min;
  beff = beff < gridDim.x ? beff : gridDim.x;
  const int blk = blockIdx.x;
  if (blk >= beff) return;
  int64_t x = (static_cast<int64_t>(blk) * total) / beff;
  const int64_t xend = (static_cast<int64_t>(blk + 1) * total) / beff;

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

  unsigned char* ktile = smem + wid * S::kTileBytes;
  unsigned char* vtile = ktile + S::kKTileBytes;
  const int vr = lane / S::kChunks;   // row within one wave load (K and V alike)
  const int vq = lane % S::kChunks;   // 16-byte chunk within the row
  const int tok_stride = hkv * D;                                  // elements per token
  const int64_t page_stride = static_cast<int64_t>(tok_stride) << page_shift;  // per page
  // byte offsets of this lane's loads inside a 16-token block of one page:
  // load i covers rows kRowsPerLoad*i .. +kRowsPerLoad-1 of the step, 16 B per lane
  int loff[S::kVLoads];
#pragma unroll
  for (int i = 0; i < S::kVLoads; ++i)
    loff[i] = 2 * ((((S::kRowsPerLoad * i) & 15) + vr) * tok_stride + 8 * vq);

  while (true) {
    const int64_t remaining = xend - x;
    const int s1 = remaining < nb - s0 ? s0 + static_cast<int>(remaining) : nb;
    const int L = uniform(clamp_len(lens[b], max_ctx));
    const int npages = (L + page - 1) >> page_shift;
    const int32_t* bt_row = bt + static_cast<int64_t>(b) * maxp;
    const int seq = b * hkv + g;

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

    // Page ids travel two steps ahead of use: the ids of step k+2 are loaded
    // (one uniform-address load per 16-token half) before the K/V loads of
    // step k+1 are issued, so every wait in the loop is satisfied in issue
    // order and the loop body stays a single basic block.
    const int sw = s0 + wid;  // this wave's first step; it takes sw, sw+4, ...
    const int nsteps = sw < s1 ? (s1 - sw + kWavesPerBlock - 1) / kWavesPerBlock : 0;
    auto step_of = [&](int k) {  // k-th step of this wave, clamped to its last one
      k = k < nsteps ? k : nsteps - 1;
      return sw + k * kWavesPerBlock;
    };
    auto load_pids = [&](int k, int& pa, int& pb) {
      const int t0 = step_of(k) * kStep;
      int ja = t0 >> page_shift, jb = (t0 + 16) >> page_shift;
      ja = ja < npages ? ja : npages - 1;
      jb = jb < npages ? jb : npages - 1;
      pa = bt_row[ja];
      pb = bt_row[jb];
    };
    auto clamp_pid = [&](int p) {
      const unsigned u = static_cast<unsigned>(uniform(p));
      return static_cast<int>(u < static_cast<unsigned>(num_pages) ? u : num_pages - 1);
    };

    auto issue = [&](int k, int pa_raw, int pb_raw, u32x4 (&kr)[S::kVLoads], u32x4 (&vv)[S::kVLoads]) {
      const int t0 = step_of(k) * kStep;
      // valid token rows in each 16-token half (0 for a step past the wave's last)
      const int live = k < nsteps ? L - t0 : 0;
      const int nA = live < 0 ? 0 : (live < 16 ? live : 16);
      const int nB = live < 16 ? 0 : (live < 32 ? live - 16 : 16);
      if constexpr (!kLanePages) {
        // pages of 16 or more tokens: each 16-token half of the step lies in one page
        const int pA = clamp_pid(pa_raw);
        const int pB = clamp_pid(pb_raw);
        const int64_t oA = pA * page_stride + static_cast<int64_t>(t0 & (page - 1)) * tok_stride;
        const int64_t oB = pB * page_stride + static_cast<int64_t>((t0 + 16) & (page - 1)) * tok_stride;
        const int bytesA = nA * tok_stride * 2, bytesB = nB * tok_stride * 2;
        const __amdgpu_buffer_rsrc_t rkA = page_rsrc(kg + oA, bytesA), rkB = page_rsrc(kg + oB, bytesB);
        const __amdgpu_buffer_rsrc_t rvA = page_rsrc(vg + oA, bytesA), rvB = page_rsrc(vg + oB, bytesB);
#pragma unroll
        for (int i = 0; i < S::kVLoads; ++i) {
          const bool hb = (S::kRowsPerLoad * i) >> 4;
          kr[i] = ld16_stream(hb ? rkB : rkA, loff[i]);
          vv[i] = ld16_stream(hb ? rvB : rvA, loff[i]);
        }
      } else {
        // small pages: every lane looks up the page of its own token
#pragma unroll
        for (int i = 0; i < S::kVLoads; ++i) {
          const int tau = S::kRowsPerLoad * i + vr;
          const int tok = t0 + tau;
          const int pg = page_at(bt_row, tok >> page_shift, npages, num_pages);
          const int64_t off = pg * page_stride + static_cast<int64_t>(tok & (page - 1)) * tok_stride + 8 * vq;
          // page_at keeps the address inside the pool; rows past the end are zeroed
          const bool ok = tok < t0 + live;
          const u32x4 zero = {0u, 0u, 0u, 0u};
          const u32x4 kv = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(kg + off));
          const u32x4 vv_ = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(vg + off));
          kr[i] = ok ? kv : zero;
          vv[i] = ok ? vv_ : zero;
        }
      }
    };

    auto compute = [&](int s, const u32x4 (&kr)[S::kVLoads], const u32x4 (&vv)[S::kVLoads]) {
      const int t0 = s * kStep;
      const bool tail = t0 + kStep > L;
      // K and V rows -> LDS (rows past the end arrived as zeros: never NaN * 0)
#pragma unroll
      for (int i = 0; i < S::kVLoads; ++i) {
        const int tau = S::kRowsPerLoad * i + vr;
        *reinterpret_cast<u32x4*>(ktile + tau * S::kKRowBytes + 16 * vq) = kr[i];
        *reinterpret_cast<u32x4*>(vtile + tau * S::kVRowBytes + 16 * vq) = vv[i];
      }
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
      // S^T = K Q^T: rows = keys 16T + 4*g4 + i, column = head c; the A operand
      // (key row c, d = 32*kk + 8*g4 .. +7) is read back from the K tile
      f32x4 sacc[2];
#pragma unroll
      for (int T = 0; T < 2; ++T) {
        sacc[T] = f32x4{0.f, 0.f, 0.f, 0.f};
        const unsigned char* krow = ktile + (16 * T + c) * S::kKRowBytes + 16 * g4;
#pragma unroll
        for (int kk = 0; kk < S::kQK; ++kk) {
          const u32x4 a = *reinterpret_cast<const u32x4*>(krow + 64 * kk);
          sacc[T] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), qop[kk],
                                                             sacc[T], 0, 0, 0);
        }
      }
      // online softmax in log2 units
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
      // O^T += V^T P^T ; V^T operand via transposed LDS reads
      const unsigned char* r0 = vtile + (4 * g4 + (c >> 2)) * S::kVRowBytes + 8 * (c & 3);
      const unsigned char* r1 = r0 + 16 * S::kVRowBytes;
#pragma unroll
      for (int dt = 0; dt < S::kDT; ++dt) {
        const i16x4 a0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(r0 + 32 * dt));
        const i16x4 a1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(r1 + 32 * dt));
        const i16x8 a = __builtin_shufflevector(a0, a1, 0, 1, 2, 3, 4, 5, 6, 7);
        acc[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), pop, acc[dt], 0,
                                                           0, 0);
      }
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    };

    // ---- this wave's steps, K/V loads one step ahead, page ids two ahead
    if (nsteps > 0) {
      u32x4 kA[S::kVLoads], vA[S::kVLoads], kB[S::kVLoads], vB[S::kVLoads];
      int pa0, pb0, pa1, pb1;
      load_pids(0, pa0, pb0);
      load_pids(1, pa1, pb1);
      issue(0, pa0, pb0, kA, vA);
      int k = 0;
      for (; k + 2 < nsteps; k += 2) {
        load_pids(k + 2, pa0, pb0);
        issue(k + 1, pa1, pb1, kB, vB);
        compute(step_of(k), kA, vA);
        load_pids(k + 3, pa1, pb1);
        issue(k + 2, pa0, pb0, kA, vA);
        compute(step_of(k + 1), kB, vB);
      }
      if (k + 1 < nsteps) {
        issue(k + 1, pa1, pb1, kB, vB);
        compute(step_of(k), kA, vA);
        compute(step_of(k + 1), kB, vB);
      } else {
        compute(step_of(k), kA, vA);
      }
    }

    // ---- combine the four waves in LDS
    float l_tot = l_lane + __shfl_xor(l_lane, 16);
    l_tot += __shfl_xor(l_tot, 32);
    f32x4* accx = reinterpret_cast<f32x4*>(smem);  // [wave][dt][lane], reuses the V tiles
    __syncthreads();  // every wave is done with its V tile
#pragma unroll
    for (int dt = 0; dt < S::kDT; ++dt) accx[(wid * S::kDT + dt) * 64 + lane] = acc[dt];
    if (g4 == 0) {
      ml_x[(wid * 16 + c) * 2 + 0] = m_run;
      ml_x[(wid * 16 + c) * 2 + 1] = l_tot;
    }
    __syncthreads();
    float mw[kWavesPerBlock], big_m = -__builtin_inff();
#pragma unroll
    for (int w = 0; w < kWavesPerBlock; ++w) {
      mw[w] = ml_x[(w * 16 + c) * 2];
      big_m = fmaxf(big_m, mw[w]);
    }
    float fw[kWavesPerBlock], den = 0.f;
#pragma unroll
    for (int w = 0; w < kWavesPerBlock; ++w) {
      // a wave with no step in this piece has m = -inf and l = 0: weight 0
      fw[w] = mw[w] == -__builtin_inff() ? 0.f : __builtin_amdgcn_exp2f(mw[w] - big_m);
      den += fw[w] * ml_x[(w * 16 + c) * 2 + 1];
    }
    const bool whole = (s0 == 0) && (s1 == nb);
    const int64_t slot = static_cast<int64_t>(blk) + seq;
    // wave wid finalises d tiles wid, wid + 4, ...
    for (int dt = wid; dt < S::kDT; dt += kWavesPerBlock) {
      f32x4 a = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int w = 0; w < kWavesPerBlock; ++w) a += fw[w] * accx[(w * S::kDT + dt) * 64 + lane];
      if (c < group) {
        if (whole) {
          const float inv = 1.0f / den;
          bf16x4 o;
#pragma unroll
          for (int i = 0; i < 4; ++i) o[i] = static_cast<__bf16>(a[i] * inv);
          uint16_t* orow = out + (static_cast<int64_t>(b) * hq + g * group + c) * D + 16 * dt + 4 * g4;
          *reinterpret_cast<u32x2*>(orow) = __builtin_bit_cast(u32x2, o);
        } else {
          float* dst = ws_acc + (slot * group + c) * D + 16 * dt + 4 * g4;
#pragma unroll
          for (int i = 0; i < 4; ++i) store_agent(dst + i, a[i]);
        }
      }
    }
    if (!whole) {
      if (wid == 0 && g4 == 0 && c < group) {
        store_agent(ws_ml + (slot * group + c) * 2 + 0, big_m);
        store_agent(ws_ml + (slot * group + c) * 2 + 1, den);
      }
      // publish this piece (every store acknowledged before the barrier),
      // count it, and let the workgroup of the last piece merge
      __builtin_amdgcn_s_waitcnt(0);
      __atomic_signal_fence(__ATOMIC_SEQ_CST);
      __syncthreads();
      const int64_t x0 = static_cast<int64_t>(pref[b]) * hkv + static_cast<int64_t>(g) * nb;
      const int64_t b0 = ((x0 + 1) * beff - 1) / total;
      const int64_t b1 = ((x0 + nb) * beff - 1) / total;
      const int pieces = static_cast<int>(b1 - b0 + 1);
      if (tid == 0)
        *flag = __hip_atomic_fetch_add(ws_cnt + seq, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) ==
                pieces - 1;
      __syncthreads();
      if (*flag) {
        const int n4 = group * D / 4;
        for (int e4 = tid; e4 < n4; e4 += kBlockThreads) {
          const int hh = (4 * e4) / D;
          float mm = -__builtin_inff(), dd = 0.f;
          f32x4 nn = {0.f, 0.f, 0.f, 0.f};
          for (int64_t pb = b0; pb <= b1; ++pb) {
            const int64_t sl = pb + seq;
            const float* mlp = ws_ml + (sl * group + hh) * 2;
            const float* ap = ws_acc + (sl * group) * D + 4 * e4;
            const f32x2 mlv = {load_agent(mlp), load_agent(mlp + 1)};
            const f32x4 av = {load_agent(ap), load_agent(ap + 1), load_agent(ap + 2), load_agent(ap + 3)};
            const float m2 = fmaxf(mm, mlv[0]);
            const float f_old = __builtin_amdgcn_exp2f(mm - m2);
            const float f_new = __builtin_amdgcn_exp2f(mlv[0] - m2);
            nn = nn * f_old + av * f_new;
            dd = dd * f_old + mlv[1] * f_new;
            mm = m2;
          }
          const float inv = 1.0f / dd;
          bf16x4 o;
#pragma unroll
          for (int i = 0; i < 4; ++i) o[i] = static_cast<__bf16>(nn[i] * inv);
          uint16_t* orow = out + (static_cast<int64_t>(b) * hq + g * group) * D + 4 * e4;
          *reinterpret_cast<u32x2*>(orow) = __builtin_bit_cast(u32x2, o);
        }
        if (tid == 0)  // ready for the next call
          __hip_atomic_store(ws_cnt + seq, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
    }
    __syncthreads();  // LDS (V tiles, exchange, flag) is reused by the next piece

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

template <int D, bool kLanePages>
static hipError_t launch_split(const LaunchArgs& a, hipStream_t st) {
  using S = Shape<D>;
  const size_t lds = static_cast<size_t>(S::kPrefOff) + static_cast<size_t>(a.batch + 1) * sizeof(int32_t);
  static bool attr_set = false;
  if (!attr_set) {
    hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&split_kernel<D, kLanePages>),
                                       hipFuncAttributeMaxDynamicSharedMemorySize, kMaxLdsBytes);
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  hipLaunchKernelGGL((split_kernel<D, kLanePages>), dim3(a.grid), dim3(kBlockThreads), lds, st,
                     a.q, a.k, a.v, a.bt, a.lens, a.out, a.ws_acc, a.ws_ml, a.ws_cnt, a.batch,
                     a.hq, a.hkv, a.group, a.page_shift, a.num_pages, a.maxp, a.min_steps,
                     a.scale * kLog2e);
  return hipGetLastError();
}

hipError_t launch_split_kernel(const LaunchArgs& a, hipStream_t st) {
  const bool lane_pages = a.page_shift < 4;
  if (a.head_dim == 128) return lane_pages ? launch_split<128, true>(a, st) : launch_split<128, false>(a, st);
  return lane_pages ? launch_split<64, true>(a, st) : launch_split<64, false>(a, st);
}

size_t split_lds_bytes(int head_dim, int batch) {
  const size_t base = head_dim == 128 ? Shape<128>::kPrefOff : Shape<64>::kPrefOff;
  return base + static_cast<size_t>(batch + 1) * sizeof(int32_t);
}

}  // namespace pda
