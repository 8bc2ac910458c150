// Paged decode attention kernels for MI355X (gfx950, CDNA4, wave64).
//
// What is computed: the paper's kernel family (iv), decode attention over a
// paged KV cache with grouped-query heads (Method, "Principle-Driven LLM
// Kernel Generator"): per sequence and kv head an online softmax over the
// cached tokens, split across many workers, then a log-sum-exp merge of the
// splits ("cross-CTA merging").  The CUDA design the paper sketches
// (m16n8k16 fragments, ldmatrix, padded shared rows, a fence-based merge) is
// prior art for another GPU; these kernels are laid out for CDNA4:
//
//  * Work split (stream-K over the context).  The flattened space of
//    (sequence b, kv-head group, 32-token step) is cut into equal contiguous
//    ranges, one per workgroup, so every workgroup moves the same amount of
//    KV whatever the length mix.  A workgroup has one wave per kv head of the
//    group (up to 8), times phases that interleave steps when there are fewer
//    than 8 kv heads: all heads of a token range are read together, so a page
//    (token rows of 2*D*Hkv bytes) is consumed in one sweep.  On MI355X this
//    access order streams at ~6.9 TB/s where independent per-head workers
//    reach ~6.0 TB/s.
//  * K and V rows are loaded with raw buffer loads (non-temporal, four
//    256-byte rows per instruction) whose descriptor is the page and covers
//    only the valid rows, so rows past the end read as zeros with no memory
//    traffic.  Loads run one step ahead of compute, page ids two steps ahead.
//  * QK^T on the matrix cores: v_mfma_f32_16x16x32_bf16 with 16 keys as A
//    rows (read back from a padded LDS tile) and the GQA query heads as B
//    columns (zero-padded to 16).  One K read serves every head of the group.
//  * The softmax runs in the MFMA result layout (lane = head column, four key
//    rows per lane), which is lane-for-lane the B operand of the P.V product.
//  * V goes through the same LDS tile and is read back transposed with
//    ds_read_b64_tr_b16 as the A operand of O^T = V^T P^T; the accumulator has
//    the head in the lane column, so the online rescale is one scalar per lane.
//  * A piece that is a whole (b, kv head) sequence is normalised and written
//    directly.  Otherwise the piece's (max in log2 units, sum, unnormalised
//    accumulator) go to a workspace slot, and merge_kernel combines them in
//    slot order (deterministic).
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <atomic>

#include "pda_internal.h"

namespace pda {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef short i16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned u32x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;

constexpr float kLog2e = 1.4426950408889634f;

// kValu: the vector-ALU variant of the step (see attn_kernel), which keeps
// one register buffer like D = 256 and reads K and V back from LDS row-wise.
template <int D, bool kValu = false>
struct Shape {
  static constexpr int kQK = D / 32;            // MFMAs per 16-key tile for QK^T
  static constexpr int kDT = D / 16;            // 16-wide d tiles of the output
  static constexpr int kChunks = D / 8;         // 16-byte chunks per key/value row
  static constexpr int kRowsPerLoad = 64 / kChunks;      // rows per wave load
  static constexpr int kLoads = kStep / kRowsPerLoad;    // loads per step (K and V each)
  // One LDS tile per wave for the K and V rows of a step, rows padded by 32
  // bytes.  Measured with SQ_LDS_BANK_CONFLICT on long70b: K rows padded by
  // 16 bytes cost 32 conflict cycles per wave step (4.2 M per call), by 32
  // none; V rows padded by 16 double them, unpadded K rows give 29 M.
  static constexpr int kKRowBytes = 2 * D + 32;
  static constexpr int kVRowBytes = 2 * D + 32;
  // D = 256 keeps one register buffer of K/V per wave (a step is 32 KB): a
  // step's K and V rows go to separate regions of the tile as soon as they
  // arrive, and the next step's loads reuse the registers.  Smaller heads
  // keep two register buffers and pass K, then V, through one region.
  static constexpr bool kOneBuffer = D == 256 || kValu;
  static constexpr int kVOffset = kOneBuffer ? kStep * kKRowBytes : 0;  // V region of the tile
  static constexpr int kTileBytes = kVOffset + kStep * kVRowBytes;
  static constexpr int kAccBytes = 64 * kDT * 16;  // one wave's accumulator in LDS
  static_assert(kAccBytes <= kTileBytes, "accumulator exchange reuses the tile");
  // The lengths read by the prefix scan stay in LDS for the pieces that
  // follow (no second global read on the way to the first page ids); at
  // D = 256 the tiles leave no room for them at the largest batch.
  static constexpr bool kLensInLds = D != 256;
};

// LDS: [waves x tile][ml exchange waves x 16 x 2 floats][prefix batch+1 ints]
// [lengths batch ints, when kLensInLds]
template <int D, bool kValu = false>
__host__ __device__ constexpr int ml_offset(int waves) { return waves * Shape<D, kValu>::kTileBytes; }
template <int D, bool kValu = false>
__host__ __device__ constexpr int pref_offset(int waves) {
  return ml_offset<D, kValu>(waves) + waves * 16 * 2 * 4;
}

__device__ __forceinline__ int uniform(int x) { return __builtin_amdgcn_readfirstlane(x); }

// Start of the first-piece stash (16-byte aligned) after `bytes` of LDS.
__host__ __device__ constexpr int stash_offset(int bytes) { return (bytes + 15) & ~15; }

// s_waitcnt vmcnt(0): wait for every outstanding vector memory load of the
// wave (expcnt 7 and lgkmcnt 15 in the gfx9 encoding mean "do not wait").
constexpr int kWaitAllVectorLoads = 0x0F70;
// s_waitcnt vmcnt(n), n < 64: vmcnt is split over bits 3:0 and 15:14.
constexpr int wait_vector_loads(int n) { return kWaitAllVectorLoads | (n & 15) | ((n >> 4) << 14); }
constexpr int kIssueK = 1, kIssueV = 2;  // which loads of a step to issue

__device__ __forceinline__ int clamp_len(int L, int max_ctx) {
  return L < 0 ? 0 : (L > max_ctx ? max_ctx : L);
}

// Key range of a sequence.  Its nq query tokens are its last nq tokens:
// query j sits at position L - nq + j and sees keys up to that position, and
// with a sliding window of W > 0 tokens only the W keys ending there.  The
// first key any query sees is seq_start; the steps of the sequence are the
// 32-token steps from the one holding seq_start to the end.
__device__ __forceinline__ int seq_start(int L, int nq, int window) {
  if (window <= 0) return 0;
  const int s = L - nq + 1 - window;
  return s > 0 ? s : 0;
}

__device__ __forceinline__ int seq_steps(int L, int nq, int window) {
  return (L + kStep - 1) / kStep - seq_start(L, nq, window) / kStep;
}

__device__ __forceinline__ u32x4 ld16(const uint16_t* p) {
  return *reinterpret_cast<const u32x4*>(p);
}

// K and V are read exactly once per call, with raw buffer loads:
//  * non-temporal (cache policy NT): on MI355X a plain streaming read runs at
//    ~7.1 TB/s this way against ~6.1 TB/s with default loads;
//  * the descriptor's base is the page (a wave-uniform 64-bit address) and
//    its size covers only the valid token rows, so rows past the end of the
//    sequence, or a step that does not exist, read as zeros without touching
//    memory.
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

// Split partials that the last workgroup to finish a sequence merges (the
// fused merge) cross workgroups on different XCDs, whose L2 caches are not
// coherent with each other.  They are stored and loaded with the
// device-coherent cache policy (sc1: stores write through, loads do not hit
// a stale line), the form the memory model gives agent-scope atomic
// accesses, so no cache-wide writeback or invalidate is needed around the
// arrival counter.
constexpr int kCachePolicyCoherent = 16;  // sc1
__device__ __forceinline__ __amdgpu_buffer_rsrc_t ws_rsrc(const float* base) {
  const uint64_t a = reinterpret_cast<uint64_t>(base);
  const uint32_t lo = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(a));
  const uint32_t hi = __builtin_amdgcn_readfirstlane(static_cast<uint32_t>(a >> 32));
  void* ub = reinterpret_cast<void*>((static_cast<uint64_t>(hi) << 32) | lo);
  return __builtin_amdgcn_make_buffer_rsrc(ub, 0, 0x7FFFFFFF, kBufferDword3);
}
__device__ __forceinline__ void store_coherent(__amdgpu_buffer_rsrc_t r, int64_t idx, f32x4 v) {
  __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, v), r, static_cast<int>(idx * 4), 0,
                                         kCachePolicyCoherent);
}
__device__ __forceinline__ void store_coherent(__amdgpu_buffer_rsrc_t r, int64_t idx, f32x2 v) {
  __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(u32x2, v), r, static_cast<int>(idx * 4), 0,
                                        kCachePolicyCoherent);
}
__device__ __forceinline__ f32x4 load_coherent4(__amdgpu_buffer_rsrc_t r, int64_t idx) {
  return __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(r, static_cast<int>(idx * 4), 0,
                                                                          kCachePolicyCoherent));
}
__device__ __forceinline__ f32x2 load_coherent2(__amdgpu_buffer_rsrc_t r, int64_t idx) {
  return __builtin_bit_cast(f32x2, __builtin_amdgcn_raw_buffer_load_b64(r, static_cast<int>(idx * 4), 0,
                                                                         kCachePolicyCoherent));
}

// Quotients on the way to the first loads of the fixed split and its
// merge.  The compiler expands a 32-bit integer division into ~25 dependent
// instructions; these divide in fp64 instead: both operands (0 <= a < 2^31,
// 0 < b < 2^31) convert exactly and the quotient a/b, correctly rounded,
// cannot reach the next integer (it is at least 1/b below it, more than the
// rounding error of a quotient below 2^31), so truncation gives
// floor(a / b).  div_small_u is the same for wave-uniform operands: the
// quotient is computed in vector registers (the scalar unit has no fp64)
// and readfirstlane returns it to scalar registers, so that nothing derived
// from it takes vector registers.  (The stream-K prologue keeps the
// compiler's integer division: there the fp64 form measured no faster and
// cost the main loop vector registers.)
__device__ __forceinline__ int div_small(int a, int b) {
  return static_cast<int>(static_cast<double>(a) / static_cast<double>(b));
}
__device__ __forceinline__ int div_small_u(int a, int b) { return uniform(div_small(a, b)); }

// Workgroup that owns flattened step x of `total`, when `parts` workgroups
// split [0, total) into ranges [w*total/parts, (w+1)*total/parts).
__device__ __forceinline__ int64_t owner_of(int64_t x, int64_t total, int64_t parts) {
  return ((x + 1) * parts - 1) / total;
}

// Value of a partner lane in the same 16-lane row (DPP), for the vector-ALU
// variant's reductions.
template <int kCtrl>
__device__ __forceinline__ float dpp_f(float x) {
  // (every source lane exists for the patterns used; bound_ctrl lets the
  // compiler fold the move into the consuming add or max as a DPP operand)
  return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(__builtin_bit_cast(int, x), kCtrl, 0xF, 0xF, true));
}
constexpr int kDppRor8 = 0x128;        // row_ror:8: lane ^ 8 within the row
constexpr int kDppHalfMirror = 0x141;  // row_half_mirror: lane ^ 7 within each half row
constexpr int kDppXor2 = 0x4E;         // quad_perm [2,3,0,1]: lane ^ 2
constexpr int kDppXor1 = 0xB1;         // quad_perm [1,0,3,2]: lane ^ 1

// Register slot of token slot `is` (0..7) in the vector-ALU variant's list of
// partial scores (index head_slot * 8 + slot): the token bit that the last
// reduce level splits comes first, the bits kept in the lane come last.
template <int NC>
__device__ __forceinline__ constexpr int valu_slot(int is) {
  return NC == 8 ? (((is & 1) << 2) | (is >> 1)) : (((is & 1) << 2) | (is & 2) | (is >> 2));
}

// The fused merge of one split sequence (kv-head group hg of sequence b,
// pieces in workgroups w0 .. w1, in slots w + base) by the workgroup that
// counted its last piece: per (query row, float4 column) of the group,
//   out = sum_j 2^(m_j - M) acc_j / sum_j 2^(m_j - M) l_j,  M = max_j m_j,
// in slot order.  When the rows x columns leave threads over, each item's
// pieces are dealt to PG groups (piece w to group (w - w0) mod PG) whose
// results are folded in group order through LDS (the tiles, free by now).
template <int D>
__device__ void merge_in_workgroup(uint16_t* __restrict__ out, const float* __restrict__ ws_acc,
                                   const float* __restrict__ ws_ml, unsigned char* smem, int b, int hg, int w0,
                                   int w1, int64_t base, int hgs, int ncols, int group, int nq, int hq) {
  constexpr int kC4 = D / 4;
  const int nthreads = blockDim.x;
  const int tid = threadIdx.x;
  const int items = hgs * ncols * kC4;
  int pgs = 1;
  while (pgs < 8 && items * pgs * 2 <= nthreads) pgs *= 2;
  const __amdgpu_buffer_rsrc_t ra = ws_rsrc(ws_acc), rm = ws_rsrc(ws_ml);
  f32x4* s_num = reinterpret_cast<f32x4*>(smem);        // [pg][item]
  f32x2* s_ml = reinterpret_cast<f32x2*>(s_num + items * pgs);
  for (int it0 = 0; it0 < items * pgs; it0 += nthreads) {
    const int it = it0 + tid;
    const bool active = it < items * pgs;
    const int item = it % items, pg = it / items;
    const int r = item / kC4, col = item - r * kC4;
    const int hi_w = r / ncols, cc = r - hi_w * ncols;
    float mm = -__builtin_inff(), ll = 0.f;
    f32x4 nn = {0.f, 0.f, 0.f, 0.f};
    if (active) {
#pragma unroll 4
      for (int w = w0 + pg; w <= w1; w += pgs) {
        const int64_t row = ((w + base) * hgs + hi_w) * ncols + cc;
        const f32x2 mlv = load_coherent2(rm, row * 2);
        const f32x4 av = load_coherent4(ra, row * D + 4 * col);
        const float m2 = fmaxf(mm, mlv[0]);
        const float mref = m2 == -__builtin_inff() ? 0.f : m2;  // pieces that saw no key
        const float fo = __builtin_amdgcn_exp2f(mm - mref);
        const float fn = __builtin_amdgcn_exp2f(mlv[0] - mref);
        nn = nn * fo + av * fn;
        ll = ll * fo + mlv[1] * fn;
        mm = m2;
      }
    }
    if (pgs > 1) {  // then items * pgs <= nthreads: one pass
      if (active) {
        s_num[it] = nn;
        s_ml[it] = f32x2{mm, ll};
      }
      __syncthreads();
      if (!active || pg != 0) continue;
      float big_m = -__builtin_inff();
      for (int p = 0; p < pgs; ++p) big_m = fmaxf(big_m, s_ml[p * items + item][0]);
      nn = f32x4{0.f, 0.f, 0.f, 0.f};
      ll = 0.f;
      for (int p = 0; p < pgs; ++p) {
        const f32x2 mlp = s_ml[p * items + item];
        const float f = mlp[0] == -__builtin_inff() ? 0.f : __builtin_amdgcn_exp2f(mlp[0] - big_m);
        nn += f * s_num[p * items + item];
        ll += f * mlp[1];
      }
    }
    if (!active) continue;
    const float inv = ll > 0.f ? 1.0f / ll : 0.f;  // a query that sees no key: zero row
    bf16x4 o;
#pragma unroll
    for (int i = 0; i < 4; ++i) o[i] = static_cast<__bf16>(nn[i] * inv);
    const int j = cc / group;
    const int h = (hg * hgs + hi_w) * group + (cc - j * group);
    *reinterpret_cast<u32x2*>(out + ((static_cast<int64_t>(b) * nq + j) * hq + h) * D + 4 * col) =
        __builtin_bit_cast(u32x2, o);
  }
}

// kFused: split sequences are merged by the last workgroup to finish each
// (plans with little partial data per sequence); otherwise merge_kernel
// runs after this kernel.
// kNC = 0: QK^T and P.V on the matrix cores (the path every entry point
// uses).  kNC = 4 or 8: the same pass with both products on the vector ALU
// (bf16 dot2 for QK^T, fp32 FMA for P.V) for up to kNC (query token, head)
// columns at D = 128 -- the measured alternative to the matrix cores,
// selected with PDA_OPT_COMPUTE_PATH.
// kFixed: the fixed split of small calls.  Workgroup w takes chunk
// w % chunks (chunk_steps steps) of the (sequence, kv-head group)
// w / chunks, known from its index alone: no steps prefix, and the length,
// q and the first page ids are requested together at entry (a small call
// is a chain of memory latencies; the prefix and the stream-K range put
// ~3 us of them before the first K/V load on MI355X).  The pieces are
// merged by merge_fixed_kernel.
template <int D, bool kLanePages, int kNC = 0, bool kFused = false, bool kFixed = false>
__global__ __launch_bounds__(64 * max_waves(D), 1) void attn_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ kc,
    const uint16_t* __restrict__ vc, const int32_t* __restrict__ bt,
    const int32_t* __restrict__ lens, uint16_t* __restrict__ out,
    float* __restrict__ ws_acc, float* __restrict__ ws_ml, int32_t* __restrict__ ws_pref,
    int32_t* __restrict__ ws_cnt, int batch, int hq, int hkv, int group, int hgs, int page_shift,
    int num_pages, int maxp, int min_steps, float scale_log2, int nq, int window, int chunks,
    int chunk_steps, int stash) {
  constexpr bool kValu = kNC > 0;
  static_assert(!kValu || (D == 128 && !kLanePages && (kNC == 4 || kNC == 8)), "vector-ALU variant shapes");
  static_assert(!kFixed || !kValu, "the fixed split runs on the matrix cores");
  // Every argument in SGPRs before anything waits on one: the compiler
  // otherwise requests them in two groups with a wait between (the second
  // group only where the first pointer is used), and since scalar loads
  // complete out of order, a wait for one of them is a wait for all, so the
  // length, page-id and q loads queued behind another round trip.  Later
  // uses of the integer arguments depend on this statement; the pointers
  // are inputs only, so their loads stay global loads.
  asm volatile(""
               : "+s"(batch), "+s"(hq), "+s"(hkv), "+s"(group), "+s"(hgs), "+s"(page_shift), "+s"(num_pages),
                 "+s"(maxp), "+s"(min_steps), "+s"(nq), "+s"(window), "+s"(chunks), "+s"(chunk_steps), "+s"(stash)
               : "s"(q), "s"(kc), "s"(vc), "s"(bt), "s"(lens), "s"(out), "s"(ws_acc), "s"(ws_ml), "s"(ws_pref));
  using S = Shape<D, kValu>;
  extern __shared__ __align__(16) unsigned char smem[];
  const int nthreads = blockDim.x;
  const int nwaves = nthreads >> 6;
  const int phases = nwaves / hgs;  // waves per kv head, interleaving steps
  const int ngroups = hkv / hgs;    // kv-head groups per sequence
  const int ncols = group * nq;     // MFMA columns in use: (query token, head of the group)
  int32_t* pref = reinterpret_cast<int32_t*>(smem + pref_offset<D, kValu>(nwaves));
  int32_t* lens_s = pref + batch + 1;  // clamped lengths (kLensInLds)
  float* ml_x = reinterpret_cast<float*>(smem + ml_offset<D, kValu>(nwaves));
  int32_t* scan = reinterpret_cast<int32_t*>(smem);  // reuses the tiles before the loop
  // stash != 0: the partial of the workgroup's first piece, when split (a
  // sequence's tail), is kept here -- [kv head of the group][column][D + 4]
  // floats after the lengths -- and written after the workgroup's last
  // piece.  Stores issued mid-kernel are waited for by the next piece's
  // first load wait (the gfx9 vector memory counter covers stores as well
  // as loads and retires them in order), so a partial written there holds
  // the next piece back until the writes are acknowledged.  Measured on the
  // 4-query-token workload (16 columns, 21 MB of partials): first-piece
  // partials skipped altogether (a timing-only build) 183 -> 175 us, kept
  // here 183 -> 178 us; the Zipf batch of 256 sequences 831 -> 825 us; the
  // others unchanged.
  float* stash_lds = reinterpret_cast<float*>(
      smem + stash_offset(pref_offset<D, kValu>(nwaves) + (batch + 1 + (S::kLensInLds ? batch : 0)) * 4));
  bool stashed = false;
  int64_t stash_row = 0;

  const int tid = threadIdx.x;
  const int page = 1 << page_shift;
  const int max_ctx = maxp << page_shift;

  if constexpr (!kFixed) {
    // ---- per-block prefix over the batch of 32-token steps per sequence ----
    // Each thread sums a run of sequences; a shuffle scan inside each wave and
    // one exchange of wave totals through LDS make the prefix with two
    // barriers (a tree over the workgroup took ~2 us of barriers).
    {
      if constexpr (S::kLensInLds) {
        // the lengths go to LDS first, read by consecutive threads with
        // several loads in flight each (a run of them read one after another
        // by its owner cost ~0.5 us per load at a batch of 8192)
  #pragma unroll 8
        for (int b = tid; b < batch; b += nthreads) lens_s[b] = clamp_len(lens[b], max_ctx);
        __syncthreads();
      }
      const int per = (batch + nthreads - 1) / nthreads;
      const int lo = tid * per;
      const int hi = min(batch, lo + per);
      int sum = 0;
      for (int b = lo; b < hi; ++b) sum += seq_steps(S::kLensInLds ? lens_s[b] : clamp_len(lens[b], max_ctx), nq, window);
      int incl = sum;  // inclusive prefix within the wave
  #pragma unroll
      for (int off = 1; off < 64; off <<= 1) {
        const int v = __shfl_up(incl, off, 64);
        if ((tid & 63) >= off) incl += v;
      }
      if ((tid & 63) == 63) scan[tid >> 6] = incl;  // wave totals
      __syncthreads();
      int before = 0;
      for (int w = 0; w < (tid >> 6); ++w) before += scan[w];
      int run = before + incl - sum;
      for (int b = lo; b < hi; ++b) {
        pref[b] = run;
        run += seq_steps(S::kLensInLds ? lens_s[b] : clamp_len(lens[b], max_ctx), nq, window);
      }
      if (tid == nthreads - 1) pref[batch] = before + incl;
      __syncthreads();
    }
    if (blockIdx.x == 0) {
      // the merge kernel reads the same prefix; empty sequences get zero rows
      // here: each wave tests 64 sequences at a time and clears the rows of the
      // empty ones together (testing one sequence after another cost ~65 ns
      // each, half a millisecond at a batch of 8192, on this workgroup alone)
      for (int b = tid; b <= batch; b += nthreads) ws_pref[b] = pref[b];
      const int row16 = nq * hq * D / 8;  // 16-byte stores per sequence
      const int ln = tid & 63;
      for (int c = (tid >> 6) * 64; c < batch; c += nwaves * 64) {
        const int bb = c + ln;
        uint64_t empty = __ballot(bb < batch && pref[bb + 1] == pref[bb]);
        while (empty) {
          const int j = __builtin_ctzll(empty);
          empty &= empty - 1;
          u32x4* orow = reinterpret_cast<u32x4*>(out + static_cast<int64_t>(c + j) * nq * hq * D);
          for (int i = ln; i < row16; i += 64) orow[i] = u32x4{0u, 0u, 0u, 0u};
        }
      }
    }
    __syncthreads();  // the scan area becomes the tiles
  }

  const int lane = tid & 63;
  const int wid = uniform(tid >> 6);  // wave-uniform: lets the compiler keep per-wave values in SGPRs
  const int hi_w = wid % hgs;         // kv head of this wave within the group
  const int ph = wid / hgs;           // step phase of this wave
  const int g4 = lane >> 4;           // lane group: MFMA k block / C row block
  const int c = lane & 15;            // MFMA row (A) / column (B, C)
  // column c = query token qj, head qh of the group (padding columns c >= ncols
  // take the last token's key range and a zero query)
  const int qj = c < ncols ? c / group : nq - 1;
  const int qh = c - (c / group) * group;
  // Vector-ALU variant: lane (vr, vq) = (lane / 16, lane % 16) holds
  // d = 8 vq .. 8 vq + 7 of token rows 4 i + vr of a step.  Its partial QK^T
  // sums over those 8 d are added across the 16 lanes of the row by a
  // transpose-reduce whose DPP partners are lane ^ 8, lane ^ 7 (within each
  // half row), lane ^ 2 and lane ^ 1, halving the values a lane holds at each
  // level.  Every lane lists heads and tokens XOR-permuted by its own lane
  // bits (vMh, vMi), chosen so that at every level the half a lane keeps is
  // the half its partner sends (no selects); at the end the lane holds the
  // whole scores of column vMh for kNC / 2 tokens of its row.
  const int vb0 = lane & 1, vb1 = (lane >> 1) & 1, vb2 = (lane >> 2) & 1, vb3 = (lane >> 3) & 1;
  const int vd3 = vb1 ^ vb2, vd4 = vb0 ^ vb2;
  const int vMh = kNC == 8 ? (vb3 << 2 | vb2 << 1 | vd3) : (vb3 << 1 | vb2);
  const int vMi = kNC == 8 ? vd4 : (vd3 | vd4 << 1);
  const int qjv = vMh < ncols ? vMh / group : nq - 1;  // query token of the lane's column

  const int blk = blockIdx.x;
  // fixed split: the piece from the workgroup index; the raw q rows of the
  // columns and the page ids of the wave's first two steps (without a
  // window they do not depend on the length) are requested before the
  // length is waited for
  int fx_b = 0, fx_hg = 0, fx_s0 = 0, fx_L = 0, fx_nb = 0, fx_w0 = 0;
  u32x4 fx_q[S::kQK];
  int fx_pa0 = 0, fx_pb0 = 0, fx_pa1 = 0, fx_pb1 = 0;
  if constexpr (kFixed) {
    const int e = div_small_u(blk, chunks);  // (sequence, kv-head group)
    fx_b = div_small_u(e, ngroups);
    fx_hg = e - fx_b * ngroups;
    fx_s0 = (blk - e * chunks) * chunk_steps;
    fx_w0 = e * chunks;  // the pair's first workgroup (and slot)
    fx_L = lens[fx_b];
    // a padding column (c >= ncols) reads a row inside q (token nq - 1,
    // head qh < group) and is zeroed where the operand is formed
    const uint16_t* qrow =
        q + ((static_cast<int64_t>(fx_b) * nq + qj) * hq + (fx_hg * hgs + hi_w) * group + qh) * D + 8 * g4;
#pragma unroll
    for (int kk = 0; kk < S::kQK; ++kk) fx_q[kk] = ld16(qrow + 32 * kk);
    if (window == 0) {
      const int32_t* bt_row = bt + static_cast<int64_t>(fx_b) * maxp;
      auto first_pids = [&](int step, int& pa, int& pb) {
        const int t0 = step * kStep;
        if constexpr (!kLanePages) {
          int ja = t0 >> page_shift, jb = (t0 + 16) >> page_shift;
          ja = ja < maxp ? ja : maxp - 1;
          jb = jb < maxp ? jb : maxp - 1;
          pa = bt_row[ja];
          pb = bt_row[jb];
        } else {
          int j = (t0 >> page_shift) + (lane & ((kStep >> page_shift) - 1));
          j = j < maxp ? j : maxp - 1;
          pa = bt_row[j];
          pb = 0;
        }
      };
      first_pids(fx_s0 + ph, fx_pa0, fx_pb0);
      first_pids(fx_s0 + ph + phases, fx_pa1, fx_pb1);
    }
    fx_nb = seq_steps(clamp_len(uniform(fx_L), max_ctx), nq, window);
    if (fx_s0 >= fx_nb) {  // a chunk past the sequence's end
      if (fx_nb == 0 && fx_s0 == 0) {
        // an empty sequence: chunk 0's workgroup writes its zero rows (the
        // heads of group fx_hg are contiguous for each query token)
        const int row16 = hgs * group * D / 8;
        for (int j = 0; j < nq; ++j) {
          u32x4* orow = reinterpret_cast<u32x4*>(
              out + ((static_cast<int64_t>(fx_b) * nq + j) * hq + fx_hg * hgs * group) * D);
          for (int i = tid; i < row16; i += nthreads) orow[i] = u32x4{0u, 0u, 0u, 0u};
        }
      }
      return;
    }
  }

  // ws_split[blk]: the (sequence, kv-head group) whose first split point
  // is this workgroup's start, else -1 -- the list of pieces to merge when
  // the batch has more sequences than workgroups (merge_kernel<.., true>)
  int32_t* ws_split = ws_pref + batch + 1;
  const int64_t total = kFixed ? 1 : static_cast<int64_t>(pref[batch]) * ngroups;
  if (!kFixed && total == 0) {
    if (tid == 0) ws_split[blk] = -1;
    return;
  }
  const int64_t per_block_min = static_cast<int64_t>(min_steps) * phases;
  int64_t beff = kFixed ? 1 : (total + per_block_min - 1) / per_block_min;
  beff = beff < gridDim.x ? beff : gridDim.x;
  if (!kFixed && blk >= beff) {
    if (tid == 0) ws_split[blk] = -1;
    return;
  }
  // a fixed-split workgroup takes one piece: steps [0, xend) from x = 0
  int64_t x = kFixed ? 0 : (static_cast<int64_t>(blk) * total) / beff;
  const int64_t xend = kFixed ? (fx_nb - fx_s0 < chunk_steps ? fx_nb - fx_s0 : chunk_steps)
                              : (static_cast<int64_t>(blk + 1) * total) / beff;

  // sequence containing step x: largest b with pref[b] * ngroups <= x
  int b = fx_b;
  if constexpr (!kFixed) {
    const int y = static_cast<int>(x / ngroups);
    int lo = 0, hi = batch - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (uniform(pref[mid]) <= y) lo = mid; else hi = mid - 1;
    }
    b = lo;
  }
  int nb = kFixed ? fx_nb : uniform(pref[b + 1]) - uniform(pref[b]);
  int rel = kFixed ? 0 : static_cast<int>(x - static_cast<int64_t>(uniform(pref[b])) * ngroups);
  int hg = kFixed ? fx_hg : rel / nb;
  int s0 = kFixed ? fx_s0 : rel - hg * nb;
  // a sequence split across workgroups w0 .. w1 is listed once, by w0 + 1
  if (!kFixed && tid == 0)
    ws_split[blk] = (s0 > 0 && owner_of(x - s0, total, beff) == blk - 1) ? b * ngroups + hg : -1;

  unsigned char* tile = smem + wid * S::kTileBytes;
  const int vr = lane / S::kChunks;   // row within one wave load (K and V alike)
  const int vq = lane % S::kChunks;   // 16-byte chunk within the row
  const int tok_stride = hkv * D;                                  // elements per token
  const int64_t page_stride = static_cast<int64_t>(tok_stride) << page_shift;  // per page
  // byte offsets of this lane's loads inside a 16-token block of one page:
  // load i covers rows kRowsPerLoad*i .. +kRowsPerLoad-1 of the step, 16 B per lane
  int loff[S::kLoads];
#pragma unroll
  for (int i = 0; i < S::kLoads; ++i)
    loff[i] = 2 * ((((S::kRowsPerLoad * i) & 15) + vr) * tok_stride + 8 * vq);

  while (true) {
    const int64_t remaining = xend - x;
    const int s1 = remaining < nb - s0 ? s0 + static_cast<int>(remaining) : nb;
    const int L = kFixed ? clamp_len(uniform(fx_L), max_ctx)
                         : uniform(S::kLensInLds ? lens_s[b] : clamp_len(lens[b], max_ctx));
    const int npages = (L + page - 1) >> page_shift;
    const int lo_seq = uniform(seq_start(L, nq, window));
    const int sb = lo_seq / kStep;                  // first step of the sequence
    // keys [lo_c, hi_c) of this lane's column; steps that cross a bound mask
    const int hi_c = L - nq + 1 + qj;
    const int lo_c = window > 0 ? max(0, hi_c - window) : 0;
    const int hi_min = L - nq + 1;                   // bound of the first query
    const int lo_max = window > 0 ? max(0, L - window) : 0;  // start of the last
    const int32_t* bt_row = bt + static_cast<int64_t>(b) * maxp;
    const int g = hg * hgs + hi_w;  // this wave's kv head

    // query operand (B of QK^T): column c, d = 32*kk + 8*g4 + e
    bf16x8 qop[S::kQK];
    if constexpr (kFixed) {
#pragma unroll
      for (int kk = 0; kk < S::kQK; ++kk)
        qop[kk] = __builtin_bit_cast(bf16x8, c < ncols ? fx_q[kk] : u32x4{0u, 0u, 0u, 0u});
    } else if constexpr (!kValu) {
      const uint16_t* qrow = q + ((static_cast<int64_t>(b) * nq + qj) * hq + g * group + qh) * D + 8 * g4;
#pragma unroll
      for (int kk = 0; kk < S::kQK; ++kk) {
        u32x4 v = {0u, 0u, 0u, 0u};
        if (c < ncols) v = ld16(qrow + 32 * kk);
        qop[kk] = __builtin_bit_cast(bf16x8, v);
      }
    }
    // vector-ALU variant: q of column hs ^ vMh at d = 8 vq .. +7, as bf16 pairs;
    // its accumulator accv[column][e] holds d = 8 vq + e over the lane's tokens
    constexpr int kNCv = kValu ? kNC : 4;  // (arrays unused on the matrix-core path)
    u32x4 qv[kNCv];
    float accv[kNCv][8];
    const int hi_v = L - nq + 1 + qjv;
    const int lo_v = window > 0 ? max(0, hi_v - window) : 0;
    if constexpr (kValu) {
#pragma unroll
      for (int hs = 0; hs < kNC; ++hs) {
        const int cq = hs ^ vMh;
        u32x4 v = {0u, 0u, 0u, 0u};
        if (cq < ncols) {
          const int jq = cq / group;
          v = ld16(q + ((static_cast<int64_t>(b) * nq + jq) * hq + g * group + (cq - jq * group)) * D +
                   8 * (lane & 15));
        }
        qv[hs] = v;
#pragma unroll
        for (int e = 0; e < 8; ++e) accv[hs][e] = 0.f;
      }
    }
    const uint16_t* kg = kc + static_cast<int64_t>(g) * D;
    const uint16_t* vg = vc + static_cast<int64_t>(g) * D;

    f32x4 acc[S::kDT];
#pragma unroll
    for (int dt = 0; dt < S::kDT; ++dt) acc[dt] = f32x4{0.f, 0.f, 0.f, 0.f};
    float m_run = -__builtin_inff();
    float l_lane = 0.f;

    // Page ids travel two steps ahead of use and K/V one step ahead, so the
    // loop body is a single basic block whose waits are met in issue order.
    // A step's loads are issued only once the previous step's have all
    // arrived: one step in flight per wave while the previous one computes
    // streams ~1% faster on MI355X than letting two steps overlap.
    const int sw = s0 + ph;  // this wave's first step; it takes sw, sw + phases, ...
    const int nsteps = sw < s1 ? (s1 - sw + phases - 1) / phases : 0;
    auto step_of = [&](int k) {  // k-th step of this wave (absolute), clamped to its last one
      k = k < nsteps ? k : nsteps - 1;
      return sb + sw + k * phases;
    };
    auto load_pids = [&](int k, int& pa, int& pb) {
      const int t0 = step_of(k) * kStep;
      if constexpr (!kLanePages) {
        // each 16-token half of the step lies in one page: two ids, wave-uniform
        int ja = t0 >> page_shift, jb = (t0 + 16) >> page_shift;
        ja = ja < npages ? ja : npages - 1;
        jb = jb < npages ? jb : npages - 1;
        pa = bt_row[ja];
        pb = bt_row[jb];
      } else {
        // pages of fewer than 16 tokens: the step spans 32 / P pages; lane l
        // holds the id of the step's page l (l mod 32 / P), read by the
        // lanes that load its rows with a lane shuffle at issue time
        int j = (t0 >> page_shift) + (lane & ((kStep >> page_shift) - 1));
        j = j < npages ? j : npages - 1;
        pa = bt_row[j];
        pb = 0;
      }
    };
    auto clamp_pid = [&](int p) {
      const unsigned u = static_cast<unsigned>(uniform(p));
      return static_cast<int>(u < static_cast<unsigned>(num_pages) ? u : num_pages - 1);
    };

    // which: kIssueK and/or kIssueV (the loads of a step, K and V interleaved
    // when both are issued together)
    auto issue = [&](int k, int pa_raw, int pb_raw, u32x4 (&kr)[S::kLoads], u32x4 (&vv)[S::kLoads],
                     int which = kIssueK | kIssueV) {
      const int t0 = step_of(k) * kStep;
      // valid token rows in each 16-token half (0 for a step past the wave's last)
      const int live = k < nsteps ? L - t0 : 0;
      // a half wholly before the first key is not read (its page may be released)
      const int nA = (live < 0 || t0 + 16 <= lo_seq) ? 0 : (live < 16 ? live : 16);
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
        if (which == (kIssueK | kIssueV)) {
#pragma unroll
          for (int i = 0; i < S::kLoads; ++i) {
            const bool hb = (S::kRowsPerLoad * i) >> 4;
            kr[i] = ld16_stream(hb ? rkB : rkA, loff[i]);
            vv[i] = ld16_stream(hb ? rvB : rvA, loff[i]);
          }
        } else if (which == kIssueK) {
#pragma unroll
          for (int i = 0; i < S::kLoads; ++i) kr[i] = ld16_stream((S::kRowsPerLoad * i) >> 4 ? rkB : rkA, loff[i]);
        } else {
#pragma unroll
          for (int i = 0; i < S::kLoads; ++i) vv[i] = ld16_stream((S::kRowsPerLoad * i) >> 4 ? rvB : rvA, loff[i]);
        }
      } else {
        // small pages: every lane takes the id of its own token's page from
        // the lane that loaded it (two steps ahead, in load_pids)
#pragma unroll
        for (int i = 0; i < S::kLoads; ++i) {
          const int tau = S::kRowsPerLoad * i + vr;
          const int tok = t0 + tau;
          const unsigned raw = static_cast<unsigned>(__shfl(pa_raw, tau >> page_shift, 64));
          const int pg = static_cast<int>(raw < static_cast<unsigned>(num_pages) ? raw : num_pages - 1);
          const int64_t off = pg * page_stride + static_cast<int64_t>(tok & (page - 1)) * tok_stride + 8 * vq;
          // the clamp keeps the address inside the pool; rows past the end
          // are replaced by zeros when staged (a select here would wait for
          // the load and serialise the step's loads)
          if (which & kIssueK) kr[i] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(kg + off));
          if (which & kIssueV) vv[i] = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(vg + off));
        }
      }
    };

    auto lds_order = [&]() {  // LDS writes of this wave before its reads, and back
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    };

    // K and V rows of the step starting at token t0 -> the tile.  V rows past
    // the end, and with a window before the first key, must be zeros, never
    // NaN * 0 in the P.V product (their scores are masked by a select, so K
    // rows need no such care on the big-page path).  With big pages, rows
    // past the end arrive as zeros (the descriptor ends there); the earlier
    // rows of the half-step that holds a window's first key are read from
    // the page, so the step that starts before that key zeroes them here
    // (a wave-uniform branch taken once per sequence piece).  With small
    // pages every dead row is selected here.
    auto live_row = [&](int t0, int i) {
      const int tok = t0 + S::kRowsPerLoad * i + vr;
      return tok < L && tok >= lo_seq;
    };
    auto stage_k = [&](const u32x4 (&kr)[S::kLoads], int t0) {
#pragma unroll
      for (int i = 0; i < S::kLoads; ++i) {
        u32x4 val = kr[i];
        if constexpr (kLanePages) val = live_row(t0, i) ? val : u32x4{0u, 0u, 0u, 0u};
        *reinterpret_cast<u32x4*>(tile + (S::kRowsPerLoad * i + vr) * S::kKRowBytes + 16 * vq) = val;
      }
    };
    auto stage_v = [&](const u32x4 (&vv_in)[S::kLoads], int t0) {
      u32x4 vv[S::kLoads];
#pragma unroll
      for (int i = 0; i < S::kLoads; ++i) {
        vv[i] = vv_in[i];
        if constexpr (kLanePages) vv[i] = live_row(t0, i) ? vv[i] : u32x4{0u, 0u, 0u, 0u};
      }
      if constexpr (!kLanePages) {
        if (t0 < lo_seq) {
#pragma unroll
          for (int i = 0; i < S::kLoads; ++i)
            vv[i] = t0 + S::kRowsPerLoad * i + vr >= lo_seq ? vv[i] : u32x4{0u, 0u, 0u, 0u};
        }
      }
#pragma unroll
      for (int i = 0; i < S::kLoads; ++i)
        *reinterpret_cast<u32x4*>(tile + S::kVOffset + (S::kRowsPerLoad * i + vr) * S::kVRowBytes + 16 * vq) =
            vv[i];
    };

    auto compute = [&](int s, const u32x4 (&kr)[S::kLoads], const u32x4 (&vv)[S::kLoads]) {
      const int t0 = s * kStep;
      const bool edge = t0 + kStep > hi_min || t0 < lo_max;  // some key of the step is masked
      if constexpr (!S::kOneBuffer) {
        stage_k(kr, t0);
        lds_order();
      }
      // S^T = K Q^T: rows = keys 16T + 4*g4 + i, column = head c; the A operand
      // is key row c, d = 32*kk + 8*g4 .. +7
      f32x4 sacc[2];
#pragma unroll
      for (int T = 0; T < 2; ++T) {
        sacc[T] = f32x4{0.f, 0.f, 0.f, 0.f};
        const unsigned char* krow = tile + (16 * T + c) * S::kKRowBytes + 16 * g4;
#pragma unroll
        for (int kk = 0; kk < S::kQK; ++kk) {
          const u32x4 a = *reinterpret_cast<const u32x4*>(krow + 64 * kk);
          sacc[T] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a), qop[kk],
                                                             sacc[T], 0, 0, 0);
        }
      }
      if constexpr (!S::kOneBuffer) {
        lds_order();
        stage_v(vv, t0);  // over the K rows just read
      }
      // online softmax in log2 units
      float sv[2][4];
      float mx = -__builtin_inff();
#pragma unroll
      for (int T = 0; T < 2; ++T)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          float v = sacc[T][i] * scale_log2;
          const int t = t0 + 16 * T + 4 * g4 + i;
          if (edge && (t >= hi_c || t < lo_c)) v = -__builtin_inff();
          sv[T][i] = v;
          mx = fmaxf(mx, v);
        }
      mx = fmaxf(mx, __shfl_xor(mx, 16));
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      const float m_new = fmaxf(m_run, mx);
      // a column that has seen no key yet keeps m = -inf: exponents then use 0
      const float m_ref = m_new == -__builtin_inff() ? 0.f : m_new;
      const float alpha = __builtin_amdgcn_exp2f(m_run - m_ref);
      m_run = m_new;
      // p = hi + lo in two bf16 operands: the P.V product then carries the
      // probabilities to ~2^-17 instead of bf16's 2^-9 (one more MFMA per d
      // tile on an otherwise idle matrix pipe)
      bf16x8 pop, pop_lo;
      float psum = 0.f;
#pragma unroll
      for (int T = 0; T < 2; ++T)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float pf = __builtin_amdgcn_exp2f(sv[T][i] - m_ref);
          const __bf16 hi = static_cast<__bf16>(pf);
          pop[4 * T + i] = hi;
          pop_lo[4 * T + i] = static_cast<__bf16>(pf - static_cast<float>(hi));
          psum += pf;
        }
      l_lane = l_lane * alpha + psum;
#pragma unroll
      for (int dt = 0; dt < S::kDT; ++dt) acc[dt] *= alpha;
      lds_order();
      // O^T += V^T P^T ; V^T operand via transposed LDS reads
      const unsigned char* r0 = tile + S::kVOffset + (4 * g4 + (c >> 2)) * S::kVRowBytes + 8 * (c & 3);
      const unsigned char* r1 = r0 + 16 * S::kVRowBytes;
#pragma unroll
      for (int dt = 0; dt < S::kDT; ++dt) {
        const i16x4 a0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(r0 + 32 * dt));
        const i16x4 a1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(r1 + 32 * dt));
        const i16x8 a = __builtin_shufflevector(a0, a1, 0, 1, 2, 3, 4, 5, 6, 7);
        const bf16x8 va = __builtin_bit_cast(bf16x8, a);
        acc[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(va, pop, acc[dt], 0, 0, 0);
        acc[dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(va, pop_lo, acc[dt], 0, 0, 0);
      }
      lds_order();
    };

    // Vector-ALU step (kValu): K and V rows are in the tile (K region, then V
    // region).  QK^T by bf16 dot2 on the lane's 8 d, the DPP transpose-reduce,
    // the online softmax on the lane's kNC / 2 scores, then the probabilities
    // and the rescale factors go through LDS (over the K rows just read) and
    // P.V is fp32 FMAs on the lane's 8 tokens x 8 d.
    auto compute_valu = [&](int s) {
      constexpr int NC = kNCv;
      constexpr int n = 8 * NC;
      constexpr int NL = NC / 2;
      const int t0 = s * kStep;
      const bool edge = t0 + kStep > hi_min || t0 < lo_max;
      // The first two reduce levels are taken as the partial sums are made:
      // head slots hs and hs + NC / 2 (the pair level 1 adds) for each token
      // slot, then two such results hs and hs + NC / 4 (the pair level 2
      // adds), re-reading the lane's K chunks from LDS for each head slot
      // pair, so that few partial sums are live at once.
      auto qk_l1 = [&](int hs, float (&t)[8]) {
#pragma unroll
        for (int is = 0; is < 8; ++is) {
          const int i = is ^ vMi;
          const u32x4 kk = *reinterpret_cast<const u32x4*>(tile + (4 * i + vr) * S::kKRowBytes + 16 * vq);
          float d0 = 0.f, d1 = 0.f;
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            // vector elements go through plain scalars: __builtin_bit_cast of
            // an element subscript (kk[j]) reads element 0 with this compiler
            const unsigned kw = kk[j], qa = qv[hs][j], qb = qv[hs + NC / 2][j];
            const bf16x2 kj = __builtin_bit_cast(bf16x2, kw);
            d0 = __builtin_amdgcn_fdot2_f32_bf16(kj, __builtin_bit_cast(bf16x2, qa), d0, false);
            d1 = __builtin_amdgcn_fdot2_f32_bf16(kj, __builtin_bit_cast(bf16x2, qb), d1, false);
          }
          t[valu_slot<NC>(is)] = d0 + dpp_f<kDppRor8>(d1);
        }
      };
      float v[n / 4];
#pragma unroll
      for (int hq = 0; hq < NC / 4; ++hq) {
        float ta[8], tb[8];
        qk_l1(hq, ta);
        qk_l1(hq + NC / 4, tb);
#pragma unroll
        for (int x = 0; x < 8; ++x) v[hq * 8 + x] = ta[x] + dpp_f<kDppHalfMirror>(tb[x]);
      }
#pragma unroll
      for (int x = 0; x < n / 8; ++x) v[x] += dpp_f<kDppXor2>(v[x + n / 8]);
#pragma unroll
      for (int x = 0; x < n / 16; ++x) v[x] += dpp_f<kDppXor1>(v[x + n / 16]);
      // v[u] = score of column vMh, token row 4 * tok(u) + vr
      auto tok = [&](int u) { return NC == 8 ? 2 * u + vd4 : 4 * u + 2 * vd4 + vd3; };
      float sv[NL];
      float mx = -__builtin_inff();
#pragma unroll
      for (int u = 0; u < NL; ++u) {
        float x = v[u] * scale_log2;
        const int t = t0 + 4 * tok(u) + vr;
        if (edge && (t >= hi_v || t < lo_v)) x = -__builtin_inff();
        sv[u] = x;
        mx = fmaxf(mx, x);
      }
      // the other lanes of the column: lane ^ 1 (and ^ 2 at NC = 4), other rows
      mx = fmaxf(mx, dpp_f<kDppXor1>(mx));
      if constexpr (NC == 4) mx = fmaxf(mx, dpp_f<kDppXor2>(mx));
      mx = fmaxf(mx, __shfl_xor(mx, 16));
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      const float m_new = fmaxf(m_run, mx);
      const float m_ref = m_new == -__builtin_inff() ? 0.f : m_new;
      const float alpha = __builtin_amdgcn_exp2f(m_run - m_ref);
      m_run = m_new;
      float psum = 0.f;
      float pv[NL];
#pragma unroll
      for (int u = 0; u < NL; ++u) {
        pv[u] = __builtin_amdgcn_exp2f(sv[u] - m_ref);
        psum += pv[u];
      }
      l_lane = l_lane * alpha + psum;
      lds_order();  // the K rows are read; p and alpha go over them
      float* pl = reinterpret_cast<float*>(tile);  // p[token row][column], then alpha[column]
#pragma unroll
      for (int u = 0; u < NL; ++u) pl[(4 * tok(u) + vr) * NC + vMh] = pv[u];
      pl[kStep * NC + vMh] = alpha;  // the same value from every lane of the column
      lds_order();
#pragma unroll
      for (int c4 = 0; c4 < NC / 4; ++c4) {
        const f32x4 al = *reinterpret_cast<const f32x4*>(pl + kStep * NC + 4 * c4);
#pragma unroll
        for (int cc = 0; cc < 4; ++cc)
#pragma unroll
          for (int e = 0; e < 8; ++e) accv[4 * c4 + cc][e] *= al[cc];
      }
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        const int tau = 4 * i + vr;
        const u32x4 vw = *reinterpret_cast<const u32x4*>(tile + S::kVOffset + tau * S::kVRowBytes + 16 * vq);
        float vf[8];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          vf[2 * j] = __builtin_bit_cast(float, vw[j] << 16);
          vf[2 * j + 1] = __builtin_bit_cast(float, vw[j] & 0xFFFF0000u);
        }
#pragma unroll
        for (int c4 = 0; c4 < NC / 4; ++c4) {
          const f32x4 pp = *reinterpret_cast<const f32x4*>(pl + tau * NC + 4 * c4);
#pragma unroll
          for (int cc = 0; cc < 4; ++cc)
#pragma unroll
            for (int e = 0; e < 8; ++e) accv[4 * c4 + cc][e] = fmaf(pp[cc], vf[e], accv[4 * c4 + cc][e]);
        }
      }
      lds_order();
    };

    // ---- this wave's steps
    if constexpr (S::kOneBuffer) {
      if (nsteps > 0) {
        u32x4 kA[S::kLoads], vA[S::kLoads];
        int pa0, pb0, pa1, pb1;
        if (kFixed && window == 0) {
          pa0 = fx_pa0, pb0 = fx_pb0, pa1 = fx_pa1, pb1 = fx_pb1;
        } else {
          load_pids(0, pa0, pb0);
          load_pids(1, pa1, pb1);
        }
        issue(0, pa0, pb0, kA, vA, kIssueK);
        issue(0, pa0, pb0, kA, vA, kIssueV);
        // A step's K rows are staged as soon as they arrive and the next
        // step's K loads reuse their registers, then the same for V: the
        // wave is never without loads in flight for a whole staging pass.
        for (int k = 0; k < nsteps; ++k) {
          load_pids(k + 2, pa0, pb0);
          // past the last step the big-page path issues zero-size loads
          // (no traffic); the small-page path would read, so it stops
          const bool next = !kLanePages || k + 1 < nsteps;
          __builtin_amdgcn_s_waitcnt(wait_vector_loads(S::kLoads));  // this step's K
          stage_k(kA, step_of(k) * kStep);
          if (next) issue(k + 1, pa1, pb1, kA, vA, kIssueK);
          __builtin_amdgcn_s_waitcnt(wait_vector_loads(S::kLoads));  // this step's V
          stage_v(vA, step_of(k) * kStep);
          lds_order();
          if (next) issue(k + 1, pa1, pb1, kA, vA, kIssueV);
          if constexpr (kValu)
            compute_valu(step_of(k));
          else
            compute(step_of(k), kA, vA);
          pa1 = pa0;
          pb1 = pb0;
        }
      }
    } else if (nsteps > 0) {
      u32x4 kA[S::kLoads], vA[S::kLoads], kB[S::kLoads], vB[S::kLoads];
      int pa0, pb0, pa1, pb1;
      if (kFixed && window == 0) {
        pa0 = fx_pa0, pb0 = fx_pb0, pa1 = fx_pa1, pb1 = fx_pb1;
      } else {
        load_pids(0, pa0, pb0);
        load_pids(1, pa1, pb1);
      }
      issue(0, pa0, pb0, kA, vA);
      int k = 0;
      // The waves of a workgroup meet at a barrier once per step, after
      // issuing the next step's loads.  Left to themselves, the older wave
      // on each SIMD wins issue arbitration and runs ahead: on MI355X waves
      // 0-3 finished long70b at ~233 us and waves 4-7 at ~306 us, so the CU
      // streamed with half its loads in flight for the last quarter.  Only
      // the steps that every wave of the workgroup has (nmin) take the
      // barrier, so each wave passes the same number of them.  (The
      // small-page path runs ~3% slower with it: its waves already wait on
      // their page-id shuffles at every issue.)
      const int nmin = kLanePages ? 0 : (s1 - s0) / phases;
      // (Small pages read their page ids with vector loads, which the wait
      // for all vector loads would also wait for: they are issued after it.)
      for (; k + 2 < nsteps; k += 2) {
        if constexpr (!kLanePages) load_pids(k + 2, pa0, pb0);
        __builtin_amdgcn_s_waitcnt(kWaitAllVectorLoads);
        issue(k + 1, pa1, pb1, kB, vB);
        if constexpr (kLanePages) load_pids(k + 2, pa0, pb0);
        if (k + 2 < nmin) __builtin_amdgcn_s_barrier();
        compute(step_of(k), kA, vA);
        if constexpr (!kLanePages) load_pids(k + 3, pa1, pb1);
        __builtin_amdgcn_s_waitcnt(kWaitAllVectorLoads);
        issue(k + 2, pa0, pb0, kA, vA);
        if constexpr (kLanePages) load_pids(k + 3, pa1, pb1);
        if (k + 2 < nmin) __builtin_amdgcn_s_barrier();
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

    if constexpr (kValu) {
      // Into the matrix-core layout that the rest of the piece expects: lane
      // (g4, c) holds d = 16 dt + 4 g4 .. +3 of column c; the four rows' token
      // partials are added here, and the column's sum l sits in g4 = 0.
      constexpr int NC = kNCv;
      float lt = l_lane + dpp_f<kDppXor1>(l_lane);
      if constexpr (NC == 4) lt += dpp_f<kDppXor2>(lt);
      lt += __shfl_xor(lt, 16);
      lt += __shfl_xor(lt, 32);
      float* xa = reinterpret_cast<float*>(tile);  // [row vr][column][D], then (m, l) per column
      float* xm = xa + 4 * NC * D;
#pragma unroll
      for (int cc = 0; cc < NC; ++cc) {
        f32x4* dst = reinterpret_cast<f32x4*>(xa + (vr * NC + cc) * D + 8 * vq);
        dst[0] = f32x4{accv[cc][0], accv[cc][1], accv[cc][2], accv[cc][3]};
        dst[1] = f32x4{accv[cc][4], accv[cc][5], accv[cc][6], accv[cc][7]};
      }
      xm[2 * vMh] = m_run;  // the same values from every lane of the column
      xm[2 * vMh + 1] = lt;
      lds_order();
#pragma unroll
      for (int dt = 0; dt < S::kDT; ++dt) {
        f32x4 sum = {0.f, 0.f, 0.f, 0.f};
        if (c < NC) {
#pragma unroll
          for (int r = 0; r < 4; ++r) sum += *reinterpret_cast<const f32x4*>(xa + (r * NC + c) * D + 16 * dt + 4 * g4);
        }
        acc[dt] = sum;
      }
      m_run = c < NC ? xm[2 * c] : -__builtin_inff();
      l_lane = (c < NC && g4 == 0) ? xm[2 * c + 1] : 0.f;
      lds_order();
    }

    // ---- finish the piece: combine the phases of each kv head, then write
    float l_tot = l_lane + __shfl_xor(l_lane, 16);
    l_tot += __shfl_xor(l_tot, 32);
    float big_m = m_run, den = l_tot;
    if (phases > 1) {
      f32x4* accx = reinterpret_cast<f32x4*>(smem);  // [wave][dt][lane], reuses the tiles
      __syncthreads();                                // every wave is done with its tile
#pragma unroll
      for (int dt = 0; dt < S::kDT; ++dt) accx[(wid * S::kDT + dt) * 64 + lane] = acc[dt];
      if (g4 == 0) {
        ml_x[(wid * 16 + c) * 2 + 0] = m_run;
        ml_x[(wid * 16 + c) * 2 + 1] = l_tot;
      }
      __syncthreads();
      if (ph == 0) {
        big_m = -__builtin_inff();
        for (int p = 0; p < phases; ++p) big_m = fmaxf(big_m, ml_x[((p * hgs + hi_w) * 16 + c) * 2]);
        den = 0.f;
#pragma unroll
        for (int dt = 0; dt < S::kDT; ++dt) acc[dt] = f32x4{0.f, 0.f, 0.f, 0.f};
        for (int p = 0; p < phases; ++p) {
          const int wp = p * hgs + hi_w;
          const float mp = ml_x[(wp * 16 + c) * 2];
          // a phase with no step in this piece has m = -inf and l = 0: weight 0
          const float f = mp == -__builtin_inff() ? 0.f : __builtin_amdgcn_exp2f(mp - big_m);
          den += f * ml_x[(wp * 16 + c) * 2 + 1];
#pragma unroll
          for (int dt = 0; dt < S::kDT; ++dt) acc[dt] += f * accx[(wp * S::kDT + dt) * 64 + lane];
        }
      }
    }
    const bool whole = (s0 == 0) && (s1 == nb);  // workgroup-uniform
    if (ph == 0 && c < ncols) {
      if (whole) {
        const float inv = den > 0.f ? 1.0f / den : 0.f;  // a query that sees no key: zero row
        uint16_t* orow = out + ((static_cast<int64_t>(b) * nq + qj) * hq + g * group + qh) * D + 4 * g4;
#pragma unroll
        for (int dt = 0; dt < S::kDT; ++dt) {
          bf16x4 o;
#pragma unroll
          for (int i = 0; i < 4; ++i) o[i] = static_cast<__bf16>(acc[dt][i] * inv);
          *reinterpret_cast<u32x2*>(orow + 16 * dt) = __builtin_bit_cast(u32x2, o);
        }
      } else {
        // slot (workgroup + sequence group) is unique: workgroup ranges are
        // contiguous; a fixed-split workgroup has one piece, in slot blk
        const int64_t slot = kFixed ? static_cast<int64_t>(blk) : static_cast<int64_t>(blk) + static_cast<int64_t>(b) * ngroups + hg;
        const int64_t row = (slot * hgs + hi_w) * ncols + c;
        if constexpr (kFused) {
          const __amdgpu_buffer_rsrc_t ra = ws_rsrc(ws_acc), rm = ws_rsrc(ws_ml);
#pragma unroll
          for (int dt = 0; dt < S::kDT; ++dt) store_coherent(ra, row * D + 4 * g4 + 16 * dt, acc[dt]);
          if (g4 == 0) store_coherent(rm, row * 2, f32x2{big_m, den});
        } else if (!kFixed && !kValu && stash && s0 > 0) {
          float* srow = stash_lds + (hi_w * ncols + c) * (D + 4);
#pragma unroll
          for (int dt = 0; dt < S::kDT; ++dt) *reinterpret_cast<f32x4*>(srow + 4 * g4 + 16 * dt) = acc[dt];
          if (g4 == 0) *reinterpret_cast<f32x2*>(srow + D) = f32x2{big_m, den};
          stashed = true;
          stash_row = row;
        } else {
          float* arow = ws_acc + row * D + 4 * g4;
#pragma unroll
          for (int dt = 0; dt < S::kDT; ++dt) *reinterpret_cast<f32x4*>(arow + 16 * dt) = acc[dt];
          if (g4 == 0) *reinterpret_cast<f32x2*>(ws_ml + row * 2) = f32x2{big_m, den};
        }
      }
    }
    if (kFused && !whole) {
      // Fused merge: every store of this piece is acknowledged (so visible
      // device-wide) before the piece is counted; the workgroup that counts
      // the sequence's last piece merges all of them in slot order, so the
      // result does not depend on the order of arrival, and resets the
      // counter for the next call (or graph replay).  The counter of a split
      // sequence is indexed by the workgroup holding its first step, which
      // no other split sequence starts in.
      __builtin_amdgcn_s_waitcnt(0);
      __syncthreads();
      int32_t* flag = reinterpret_cast<int32_t*>(ml_x);
      int w0, w1;
      if constexpr (kFixed) {  // the pair's chunks that hold steps: workgroups w0 .. w0 + n - 1
        w0 = fx_w0;
        w1 = fx_w0 + div_small_u(nb + chunk_steps - 1, chunk_steps) - 1;
      } else {
        const int64_t x0 = static_cast<int64_t>(pref[b]) * ngroups + static_cast<int64_t>(hg) * nb;
        w0 = static_cast<int>(owner_of(x0, total, beff));
        w1 = static_cast<int>(owner_of(x0 + nb - 1, total, beff));
      }
      if (tid == 0)
        *flag = __hip_atomic_fetch_add(ws_cnt + w0, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == w1 - w0;
      __syncthreads();
      if (uniform(*flag)) {
        merge_in_workgroup<D>(out, ws_acc, ws_ml, smem, b, hg, w0, w1,
                              kFixed ? 0 : static_cast<int64_t>(b) * ngroups + hg, hgs, ncols, group, nq, hq);
        if (tid == 0) __hip_atomic_store(ws_cnt + w0, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
      __syncthreads();  // the flag and the tiles are reused by the next piece
    } else if (phases > 1) {
      __syncthreads();  // the exchange area is a tile again
    }

    x += s1 - s0;
    if (x >= xend) {
      if (!kFixed && !kValu && stashed) {  // the first piece's partial, kept in LDS (same lanes as wrote it)
        const float* srow = stash_lds + (hi_w * ncols + c) * (D + 4);
        float* arow = ws_acc + stash_row * D + 4 * g4;
#pragma unroll
        for (int dt = 0; dt < S::kDT; ++dt)
          *reinterpret_cast<f32x4*>(arow + 16 * dt) = *reinterpret_cast<const f32x4*>(srow + 4 * g4 + 16 * dt);
        if (g4 == 0) *reinterpret_cast<f32x2*>(ws_ml + stash_row * 2) = *reinterpret_cast<const f32x2*>(srow + D);
      }
      break;
    }
    s0 = 0;
    if (++hg == ngroups) {
      hg = 0;
      do {
        ++b;
        nb = uniform(pref[b + 1]) - uniform(pref[b]);
      } while (nb == 0);
    }
  }
}

// Merge of split pieces: one workgroup per (sequence, kv-head group, chunk
// of its query heads).  Per query head:
//   out = sum_j 2^(m_j - M) acc_j / sum_j 2^(m_j - M) l_j,  M = max_j m_j,
// over the pieces in slot order.  Threads split (head of the chunk, group of
// pieces, float4 column); kPG piece groups are folded through LDS.  kPG = 8
// suits plans where a sequence spans many workgroups (long contexts), kPG = 1
// plans where it spans a few (then a workgroup covers more heads).
// kBySplit: the grid runs over the attention workgroups instead of the
// sequences, workgroup j merging the sequence listed in ws_split[j] (if
// any), for batches with more sequences than attention workgroups, where
// most sequences are whole and a grid over all of them only returns.
template <int D, int kPG, bool kBySplit = false>
__global__ __launch_bounds__(kMergeThreads) void merge_kernel(
    uint16_t* __restrict__ out, const float* __restrict__ ws_acc, const float* __restrict__ ws_ml,
    const int32_t* __restrict__ ws_pref, int batch, int hq, int hkv, int group, int hgs, int min_steps,
    int phases, int grid_blocks, int nq) {
  constexpr int kCols = D / 4;
  constexpr int kHPB = kMergeThreads / (kPG * kCols);  // query heads per workgroup
  static_assert(kHPB >= 1 && kHPB * kPG * kCols == kMergeThreads, "merge layout");
  __shared__ f32x4 s_num[kHPB][kPG][kCols];
  __shared__ float s_m[kHPB][kPG], s_l[kHPB][kPG];

  const int ngroups = hkv / hgs;
  const int ncols = group * nq;   // (query token, head) columns per kv head
  const int heads = hgs * ncols;  // query rows of one kv-head group
  const int chunks = (heads + kHPB - 1) / kHPB;
  int e = blockIdx.x / chunks;
  const int chunk = blockIdx.x - e * chunks;
  if constexpr (kBySplit) {
    e = ws_pref[batch + 1 + e];  // ws_split
    if (e < 0) return;
  }
  const int b = e / ngroups;
  const int hg = e - b * ngroups;
  // The three prefix entries are requested together and the one early
  // return needs all of them (with a return on nb == 0 first, the total
  // was requested only once nb had arrived: one more dependent load).
  const int pb0 = ws_pref[b], pb1 = ws_pref[b + 1], pbt = ws_pref[batch];
  const int nb = pb1 - pb0;
  int64_t total = static_cast<int64_t>(pbt) * ngroups;
  total = total > 0 ? total : 1;  // an all-empty batch returns below (nb == 0)
  const int64_t per_block_min = static_cast<int64_t>(min_steps) * phases;
  int64_t beff = (total + per_block_min - 1) / per_block_min;
  beff = beff < grid_blocks ? beff : grid_blocks;
  const int64_t x0 = static_cast<int64_t>(pb0) * ngroups + static_cast<int64_t>(hg) * nb;
  const int64_t w0 = owner_of(x0, total, beff);
  const int64_t w1 = owner_of(x0 + (nb > 0 ? nb : 1) - 1, total, beff);
  // an empty sequence (its zero row written by the attention kernel), or one
  // that a single workgroup covered and wrote
  if (nb == 0 || w0 == w1) return;

  const int tid = threadIdx.x;
  const int hs = tid / (kPG * kCols);
  const int pg = (tid / kCols) % kPG;
  const int col = tid % kCols;
  const int hh = chunk * kHPB + hs;  // query head within the kv-head group
  const bool active = hh < heads;
  const int64_t base = static_cast<int64_t>(b) * ngroups + hg;
  float mm = -__builtin_inff(), ll = 0.f;
  f32x4 nn = {0.f, 0.f, 0.f, 0.f};
  if (active) {
    const int hi_w = hh / ncols, c = hh - (hh / ncols) * ncols;
#pragma unroll 4
    for (int64_t w = w0 + pg; w <= w1; w += kPG) {
      const int64_t row = ((w + base) * hgs + hi_w) * ncols + c;
      const f32x2 mlv = *reinterpret_cast<const f32x2*>(ws_ml + row * 2);
      const f32x4 av = *reinterpret_cast<const f32x4*>(ws_acc + row * D + 4 * col);
      const float m2 = fmaxf(mm, mlv[0]);
      const float mref = m2 == -__builtin_inff() ? 0.f : m2;  // pieces that saw no key
      const float fo = __builtin_amdgcn_exp2f(mm - mref);
      const float fn = __builtin_amdgcn_exp2f(mlv[0] - mref);
      nn = nn * fo + av * fn;
      ll = ll * fo + mlv[1] * fn;
      mm = m2;
    }
  }
  if (kPG > 1) {
    s_num[hs][pg][col] = nn;
    if (col == 0) {
      s_m[hs][pg] = mm;
      s_l[hs][pg] = ll;
    }
    __syncthreads();
    if (pg != 0) return;
    float big_m = -__builtin_inff();
#pragma unroll
    for (int p = 0; p < kPG; ++p) big_m = fmaxf(big_m, s_m[hs][p]);
    float den = 0.f;
    f32x4 num = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int p = 0; p < kPG; ++p) {
      // a piece group that got no piece has m = -inf: weight 0
      const float f = s_m[hs][p] == -__builtin_inff() ? 0.f : __builtin_amdgcn_exp2f(s_m[hs][p] - big_m);
      den += f * s_l[hs][p];
      num += f * s_num[hs][p][col];
    }
    nn = num;
    ll = den;
  }
  if (!active) return;
  const float inv = ll > 0.f ? 1.0f / ll : 0.f;  // a query that sees no key: zero row
  bf16x4 o;
#pragma unroll
  for (int i = 0; i < 4; ++i) o[i] = static_cast<__bf16>(nn[i] * inv);
  const int hi_w = hh / ncols, c = hh - hi_w * ncols;
  const int j = c / group;
  const int h = (hg * hgs + hi_w) * group + (c - j * group);
  *reinterpret_cast<u32x2*>(out + ((static_cast<int64_t>(b) * nq + j) * hq + h) * D + 4 * col) =
      __builtin_bit_cast(u32x2, o);
}

// Merge of the fixed split: the pieces of (sequence b, kv-head group hg) are
// the slots e * chunks + w, w < n, with e = b * groups + hg and n the number
// of chunk_steps-step chunks the sequence's steps fill.  n follows from the
// length alone, so the partials of every chunk are requested together with
// the length and those of chunks past n (stale data of other calls) are
// selected away.  n = 1: the attention kernel wrote the sequence itself,
// and n = 0 its zero row.  Same layout and slot order as merge_kernel.
template <int D, int kPG>
__global__ __launch_bounds__(kMergeThreads) void merge_fixed_kernel(
    uint16_t* __restrict__ out, const float* __restrict__ ws_acc, const float* __restrict__ ws_ml,
    const int32_t* __restrict__ lens, int hq, int hkv, int group, int hgs, int nq, int window, int max_ctx,
    int chunks, int chunk_steps) {
  constexpr int kCols = D / 4;
  constexpr int kHPB = kMergeThreads / (kPG * kCols);  // query heads per workgroup
  static_assert(kHPB >= 1 && kHPB * kPG * kCols == kMergeThreads, "merge layout");
  __shared__ f32x4 s_num[kHPB][kPG][kCols];
  __shared__ float s_m[kHPB][kPG], s_l[kHPB][kPG];

  // one round trip for the arguments: this statement needs all of them in
  // SGPRs and every later use of an integer argument depends on it
  // (pointers are inputs only, so their loads stay global loads)
  asm volatile(""
               : "+s"(hq), "+s"(hkv), "+s"(group), "+s"(hgs), "+s"(nq), "+s"(window), "+s"(max_ctx), "+s"(chunks),
                 "+s"(chunk_steps)
               : "s"(out), "s"(ws_acc), "s"(ws_ml), "s"(lens));
  const int ngroups = div_small_u(hkv, hgs);
  const int ncols = group * nq;
  const int heads = hgs * ncols;
  const int hchunks = (heads + kHPB - 1) / kHPB;
  const int e = div_small_u(static_cast<int>(blockIdx.x), hchunks);
  const int chunk = blockIdx.x - e * hchunks;
  const int b = div_small_u(e, ngroups);
  const int hg = e - b * ngroups;
  const int len = lens[b];

  const int tid = threadIdx.x;
  const int hs = tid / (kPG * kCols);
  const int pg = (tid / kCols) % kPG;
  const int col = tid % kCols;
  const int hh = chunk * kHPB + hs;  // query head within the kv-head group
  const bool active = hh < heads;
  const int hhc = active ? hh : 0;    // (a thread past the heads reads a valid row and writes nothing)
  const int hi_w = div_small(hhc, ncols), c = hhc - hi_w * ncols;
  auto row_of = [&](int w) { return ((static_cast<int64_t>(e) * chunks + w) * hgs + hi_w) * ncols + c; };
  // the first kAhead pieces of this thread's piece group, requested before
  // the length is waited for (clamped into the sequence's own slots)
  constexpr int kAhead = 4;
  f32x2 mla[kAhead];
  f32x4 aca[kAhead];
#pragma unroll
  for (int i = 0; i < kAhead; ++i) {
    const int w = pg + i * kPG < chunks ? pg + i * kPG : chunks - 1;
    mla[i] = *reinterpret_cast<const f32x2*>(ws_ml + row_of(w) * 2);
    aca[i] = *reinterpret_cast<const f32x4*>(ws_acc + row_of(w) * D + 4 * col);
  }
  __builtin_amdgcn_sched_barrier(0);  // every load above issues before the length is used
  const int nb = seq_steps(clamp_len(len, max_ctx), nq, window);
  const int n = div_small_u(nb + chunk_steps - 1, chunk_steps);  // pieces: slots e * chunks + [0, n)
  float mm = -__builtin_inff(), ll = 0.f;
  f32x4 nn = {0.f, 0.f, 0.f, 0.f};
  auto take = [&](float mj, float lj, f32x4 aj) {
    const float m2 = fmaxf(mm, mj);
    const float mref = m2 == -__builtin_inff() ? 0.f : m2;  // no piece yet, or one that saw no key
    const float fo = __builtin_amdgcn_exp2f(mm - mref);
    const float fn = __builtin_amdgcn_exp2f(mj - mref);
    nn = nn * fo + aj * fn;
    ll = ll * fo + lj * fn;
    mm = m2;
  };
#pragma unroll
  for (int i = 0; i < kAhead; ++i) {
    const bool use = pg + i * kPG < n;  // a piece of this call (else stale data, selected away)
    take(use ? mla[i][0] : -__builtin_inff(), use ? mla[i][1] : 0.f, use ? aca[i] : f32x4{0.f, 0.f, 0.f, 0.f});
  }
  for (int w = pg + kAhead * kPG; w < n; w += kPG) {
    const f32x2 mlv = *reinterpret_cast<const f32x2*>(ws_ml + row_of(w) * 2);
    take(mlv[0], mlv[1], *reinterpret_cast<const f32x4*>(ws_acc + row_of(w) * D + 4 * col));
  }
  if (n <= 1) return;  // whole or empty: written by the attention kernel (uniform per workgroup)
  if (kPG > 1) {
    s_num[hs][pg][col] = nn;
    if (col == 0) {
      s_m[hs][pg] = mm;
      s_l[hs][pg] = ll;
    }
    __syncthreads();
    if (pg != 0) return;
    float big_m = -__builtin_inff();
#pragma unroll
    for (int p = 0; p < kPG; ++p) big_m = fmaxf(big_m, s_m[hs][p]);
    float den = 0.f;
    f32x4 num = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int p = 0; p < kPG; ++p) {
      const float f = s_m[hs][p] == -__builtin_inff() ? 0.f : __builtin_amdgcn_exp2f(s_m[hs][p] - big_m);
      den += f * s_l[hs][p];
      num += f * s_num[hs][p][col];
    }
    nn = num;
    ll = den;
  }
  if (!active) return;
  const float inv = ll > 0.f ? 1.0f / ll : 0.f;  // an empty sequence, or a query that sees no key: zero row
  bf16x4 o;
#pragma unroll
  for (int i = 0; i < 4; ++i) o[i] = static_cast<__bf16>(nn[i] * inv);
  const int j = div_small(c, group);
  const int h = (hg * hgs + hi_w) * group + (c - j * group);
  *reinterpret_cast<u32x2*>(out + ((static_cast<int64_t>(b) * nq + j) * hq + h) * D + 4 * col) =
      __builtin_bit_cast(u32x2, o);
}

template <int D, bool kLanePages, int kNC = 0, bool kFused = false, bool kFixed = false>
static hipError_t launch_attn(const LaunchArgs& a, hipStream_t st) {
  const size_t lds = a.stash ? attn_stash_lds_bytes(D, a.batch, a.waves, a.hgs, a.group * a.nq, kNC > 0)
                             : attn_lds_bytes(D, a.batch, a.waves, kNC > 0);
  // the dynamic-LDS limit is raised once per device (bit = device ordinal)
  static std::atomic<uint64_t> attr_set{0};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  const uint64_t bit = dev < 64 ? uint64_t{1} << dev : 0;
  if (!bit || !(attr_set.load() & bit)) {
    e = hipFuncSetAttribute(reinterpret_cast<const void*>(&attn_kernel<D, kLanePages, kNC, kFused, kFixed>),
                            hipFuncAttributeMaxDynamicSharedMemorySize, kMaxLdsBytes);
    if (e != hipSuccess) return e;
    attr_set.fetch_or(bit);
  }
  hipLaunchKernelGGL((attn_kernel<D, kLanePages, kNC, kFused, kFixed>), dim3(a.grid), dim3(64 * a.waves), lds, st, a.q,
                     a.k, a.v, a.bt, a.lens, a.out, a.ws_acc, a.ws_ml, a.ws_pref, a.ws_cnt, a.batch, a.hq, a.hkv,
                     a.group, a.hgs, a.page_shift, a.num_pages, a.maxp, a.min_steps, a.scale * kLog2e, a.nq,
                     a.window, a.chunks, a.chunk_steps, a.stash ? 1 : 0);
  return hipGetLastError();
}

hipError_t launch_attn_kernel(const LaunchArgs& a, hipStream_t st) {
  const bool lane_pages = a.page_shift < 4;
  if (a.waves > max_waves(a.head_dim)) return hipErrorInvalidValue;
  if (a.valu_cols) {
    // vector-ALU variant: D = 128, pages of 16 tokens or more, at most 8 columns, merge kernel
    if (a.head_dim != 128 || lane_pages || a.group * a.nq > a.valu_cols || a.fused || a.chunks > 0)
      return hipErrorInvalidValue;
    return a.valu_cols == 4 ? launch_attn<128, false, 4>(a, st) : launch_attn<128, false, 8>(a, st);
  }
  if (a.chunks > 0 && a.fused) {
    if (a.head_dim == 128)
      return lane_pages ? launch_attn<128, true, 0, true, true>(a, st) : launch_attn<128, false, 0, true, true>(a, st);
    if (a.head_dim == 256)
      return lane_pages ? launch_attn<256, true, 0, true, true>(a, st) : launch_attn<256, false, 0, true, true>(a, st);
    return lane_pages ? launch_attn<64, true, 0, true, true>(a, st) : launch_attn<64, false, 0, true, true>(a, st);
  }
  if (a.chunks > 0) {
    if (a.head_dim == 128)
      return lane_pages ? launch_attn<128, true, 0, false, true>(a, st) : launch_attn<128, false, 0, false, true>(a, st);
    if (a.head_dim == 256)
      return lane_pages ? launch_attn<256, true, 0, false, true>(a, st) : launch_attn<256, false, 0, false, true>(a, st);
    return lane_pages ? launch_attn<64, true, 0, false, true>(a, st) : launch_attn<64, false, 0, false, true>(a, st);
  }
  if (a.fused) {
    if (a.head_dim == 128)
      return lane_pages ? launch_attn<128, true, 0, true>(a, st) : launch_attn<128, false, 0, true>(a, st);
    if (a.head_dim == 256)
      return lane_pages ? launch_attn<256, true, 0, true>(a, st) : launch_attn<256, false, 0, true>(a, st);
    return lane_pages ? launch_attn<64, true, 0, true>(a, st) : launch_attn<64, false, 0, true>(a, st);
  }
  if (a.head_dim == 128) return lane_pages ? launch_attn<128, true>(a, st) : launch_attn<128, false>(a, st);
  if (a.head_dim == 256) return lane_pages ? launch_attn<256, true>(a, st) : launch_attn<256, false>(a, st);
  return lane_pages ? launch_attn<64, true>(a, st) : launch_attn<64, false>(a, st);
}

template <int D, int kPG, bool kBySplit = false>
static hipError_t launch_merge(const LaunchArgs& a, hipStream_t st) {
  constexpr int kHPB = kMergeThreads / (kPG * (D / 4));
  const int heads = a.hgs * a.group * a.nq;
  const int chunks = (heads + kHPB - 1) / kHPB;
  const dim3 grid((kBySplit ? a.grid : a.batch * (a.hkv / a.hgs)) * chunks);
  hipLaunchKernelGGL((merge_kernel<D, kPG, kBySplit>), grid, dim3(kMergeThreads), 0, st, a.out, a.ws_acc, a.ws_ml,
                     a.ws_pref, a.batch, a.hq, a.hkv, a.group, a.hgs, a.min_steps, a.waves / a.hgs, a.grid,
                     a.nq);
  return hipGetLastError();
}

template <int D, int kPG>
static hipError_t launch_merge_fixed(const LaunchArgs& a, hipStream_t st) {
  constexpr int kHPB = kMergeThreads / (kPG * (D / 4));
  const int heads = a.hgs * a.group * a.nq;
  const int hchunks = (heads + kHPB - 1) / kHPB;
  const dim3 grid(a.batch * (a.hkv / a.hgs) * hchunks);
  hipLaunchKernelGGL((merge_fixed_kernel<D, kPG>), grid, dim3(kMergeThreads), 0, st, a.out, a.ws_acc, a.ws_ml, a.lens,
                     a.hq, a.hkv, a.group, a.hgs, a.nq, a.window, a.maxp << a.page_shift, a.chunks, a.chunk_steps);
  return hipGetLastError();
}

hipError_t launch_merge_kernel(const LaunchArgs& a, hipStream_t st) {
  if (a.chunks > 0) {
    // several pieces per sequence: piece groups folded through LDS
    const bool many = a.chunks >= 8;
    if (a.head_dim == 128) return many ? launch_merge_fixed<128, 8>(a, st) : launch_merge_fixed<128, 1>(a, st);
    if (a.head_dim == 256) return many ? launch_merge_fixed<256, 4>(a, st) : launch_merge_fixed<256, 1>(a, st);
    return many ? launch_merge_fixed<64, 8>(a, st) : launch_merge_fixed<64, 1>(a, st);
  }
  // expected pieces per split sequence: workgroups per kv-head-group sequence
  const int64_t seqs = static_cast<int64_t>(a.batch) * (a.hkv / a.hgs);
  const bool many = a.grid >= 8 * seqs;
  // more sequences than attention workgroups: at most one split sequence
  // per workgroup boundary, listed by the attention kernel
  const bool by_split = seqs > a.grid;
  if (a.head_dim == 128)
    return many ? launch_merge<128, 8>(a, st) : by_split ? launch_merge<128, 1, true>(a, st) : launch_merge<128, 1>(a, st);
  if (a.head_dim == 256)
    return many ? launch_merge<256, 4>(a, st) : by_split ? launch_merge<256, 1, true>(a, st) : launch_merge<256, 1>(a, st);
  return many ? launch_merge<64, 8>(a, st) : by_split ? launch_merge<64, 1, true>(a, st) : launch_merge<64, 1>(a, st);
}

size_t attn_stash_lds_bytes(int head_dim, int batch, int waves, int hgs, int cols, bool valu) {
  return static_cast<size_t>(stash_offset(static_cast<int>(attn_lds_bytes(head_dim, batch, waves, valu)))) +
         static_cast<size_t>(hgs) * cols * (head_dim + 4) * sizeof(float);
}

size_t attn_lds_bytes(int head_dim, int batch, int waves, bool valu) {
  const int base = head_dim == 256   ? pref_offset<256>(waves)
                   : head_dim == 128 ? (valu ? pref_offset<128, true>(waves) : pref_offset<128>(waves))
                                     : pref_offset<64>(waves);
  const bool lens_in_lds = head_dim == 256 ? Shape<256>::kLensInLds : Shape<128>::kLensInLds;
  return static_cast<size_t>(base) + static_cast<size_t>(batch + 1 + (lens_in_lds ? batch : 0)) * sizeof(int32_t);
}

}  // namespace pda
