// C-ABI host side of the paged decode attention library: argument checks
// (before any HIP call), the split planner, per-(device, stream) workspaces
// and optional event timing.  The kernels live in pda_kernels.hip.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <climits>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <map>
#include <mutex>
#include <string>
#include <utility>
#include <vector>

#include "pda.h"
#include "pda_append.h"
#include "pda_probe.h"
#include "pda_gemv.h"
#include "pda_internal.h"

namespace {

thread_local std::string g_err;

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

int hip_fail(hipError_t e, const char* what) {
  return fail(PDA_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

int env_int(const char* name, int dflt, int lo, int hi) {
  const char* s = std::getenv(name);
  if (!s || !*s) return dflt;
  long v = std::strtol(s, nullptr, 10);
  if (v < lo) v = lo;
  if (v > hi) v = hi;
  return static_cast<int>(v);
}

// Tunables of the planner: defaults, environment overrides, pda_set_option.
constexpr int kMaxBlocksPerCu = 8;
constexpr int kMaxMinSteps = 1 << 30;
std::atomic<int> g_blocks_per_cu{-1};
std::atomic<int> g_min_steps{-1};
std::atomic<int> g_compute_path{-1};
std::atomic<int> g_fused_merge{-1};
std::atomic<int> g_kv_group{-1};
std::atomic<int> g_fixed_split{-1};

int blocks_per_cu() {
  int v = g_blocks_per_cu.load();
  if (v < 0) {
    v = env_int("PDA_BLOCKS_PER_CU", 1, 1, kMaxBlocksPerCu);
    g_blocks_per_cu.store(v);
  }
  return v;
}
// Fewest 32-token steps per wave the caller fixed (0 = the planner's choice).
int min_steps_option() {
  int v = g_min_steps.load();
  if (v < 0) {
    v = env_int("PDA_MIN_STEPS", 0, 0, kMaxMinSteps);
    g_min_steps.store(v);
  }
  return v;
}

int compute_path() {
  int v = g_compute_path.load();
  if (v < 0) {
    v = env_int("PDA_COMPUTE_PATH", 0, 0, 1);
    g_compute_path.store(v);
  }
  return v;
}

int fused_merge() {
  int v = g_fused_merge.load();
  if (v < 0) {
    v = env_int("PDA_FUSED_MERGE", 0, 0, 2);
    g_fused_merge.store(v);
  }
  return v;
}

// Most kv heads one attention workgroup reads together (0 = the plan's own choice).
int kv_group_cap() {
  int v = g_kv_group.load();
  if (v < 0) {
    v = env_int("PDA_KV_GROUP", 0, 0, pda::kMaxWaves);
    g_kv_group.store(v);
  }
  return v;
}

// 1 (default): latency-bound calls take the fixed split; 0: every call
// takes the stream-K split.
int fixed_split() {
  int v = g_fixed_split.load();
  if (v < 0) {
    v = env_int("PDA_FIXED_SPLIT", 1, 0, 1);
    g_fixed_split.store(v);
  }
  return v;
}

bool is_pow2(int x) { return x > 0 && (x & (x - 1)) == 0; }
int log2i(int x) {
  int s = 0;
  while ((1 << s) < x) ++s;
  return s;
}

int check_shape(int32_t batch, int32_t hq, int32_t hkv, int32_t d, int32_t p, int32_t maxp) {
  if (batch < 0) return fail(PDA_ERR_SHAPE, "batch must be >= 0 (got %d)", batch);
  if (hq <= 0 || hkv <= 0) return fail(PDA_ERR_SHAPE, "head counts must be positive (q %d, kv %d)", hq, hkv);
  if (hq % hkv) return fail(PDA_ERR_SHAPE, "num_q_heads %d is not a multiple of num_kv_heads %d", hq, hkv);
  if (hkv > PDA_MAX_KV_HEADS)
    return fail(PDA_ERR_UNSUPPORTED, "num_kv_heads %d exceeds %d", hkv, PDA_MAX_KV_HEADS);
  if (hq / hkv > PDA_MAX_GROUP)
    return fail(PDA_ERR_UNSUPPORTED, "query group %d exceeds %d", hq / hkv, PDA_MAX_GROUP);
  if (d != 64 && d != 128 && d != 256) return fail(PDA_ERR_UNSUPPORTED, "head_dim %d (supported: 64, 128, 256)", d);
  if (p <= 0 || maxp <= 0) return fail(PDA_ERR_SHAPE, "page_size and max_pages_per_seq must be positive");
  if (!is_pow2(p) || p > PDA_MAX_PAGE_SIZE)
    return fail(PDA_ERR_UNSUPPORTED, "page_size %d (supported: powers of two up to %d)", p, PDA_MAX_PAGE_SIZE);
  if (batch > PDA_MAX_BATCH) return fail(PDA_ERR_UNSUPPORTED, "batch %d exceeds %d", batch, PDA_MAX_BATCH);
  const int64_t max_ctx = static_cast<int64_t>(maxp) * p;
  if (max_ctx > (int64_t{1} << 30)) return fail(PDA_ERR_SHAPE, "max_pages_per_seq * page_size too large");
  const int64_t steps = static_cast<int64_t>(batch) * ((max_ctx + pda::kStep - 1) / pda::kStep);
  if (steps >= (int64_t{1} << 31))
    return fail(PDA_ERR_UNSUPPORTED, "batch * max context exceeds 2^36 tokens");
  return PDA_OK;
}

// Attention-only limits on top of check_shape.
int check_attention(int32_t batch, int32_t hq, int32_t hkv, int32_t d, int32_t p, int32_t maxp) {
  int rc = check_shape(batch, hq, hkv, d, p, maxp);
  if (rc) return rc;
  if (d == 256 && batch > PDA_MAX_BATCH_D256)
    return fail(PDA_ERR_UNSUPPORTED, "batch %d exceeds %d at head_dim 256", batch, PDA_MAX_BATCH_D256);
  return PDA_OK;
}

// The compute path's own limits (PDA_OPT_COMPUTE_PATH): the vector-ALU
// variant takes D = 128, pages of >= 16 tokens and <= 8 columns, and its LDS
// tiles bound the batch.  *valu_cols = 0 (matrix cores) or 4 / 8.
int check_compute_path(int32_t d, int32_t p, int cols, int32_t batch, int* valu_cols) {
  *valu_cols = 0;
  if (compute_path() != 1) return PDA_OK;
  if (d != 128 || p < 16 || cols > 8)
    return fail(PDA_ERR_UNSUPPORTED,
                "the vector-ALU compute path takes head_dim 128, page_size >= 16 and at most 8 columns "
                "(got head_dim %d, page_size %d, %d columns)", d, p, cols);
  if (pda::attn_lds_bytes(d, batch, pda::max_waves(d), true) > static_cast<size_t>(pda::kMaxLdsBytes))
    return fail(PDA_ERR_UNSUPPORTED, "batch %d needs more LDS than a workgroup has on the vector-ALU path", batch);
  *valu_cols = cols <= 4 ? 4 : 8;
  return PDA_OK;
}

struct Plan {
  int grid = 0;
  int waves = 0;   // per workgroup
  int hgs = 0;     // kv heads per workgroup
  int min_steps = 0;   // fewest 32-token steps per wave
  bool fused = false;  // split sequences merged by their last workgroup
  int chunks = 0;       // > 0: fixed split, chunks per (sequence, kv-head group)
  int chunk_steps = 0;  // 32-token steps per chunk of the fixed split
  int64_t slots = 0;
  int64_t off_acc = 0, off_ml = 0, off_pref = 0, bytes = 0;
};

int64_t align256(int64_t x) { return (x + 255) & ~int64_t{255}; }

// Largest divisor of hkv that is at most max_waves: the kv heads a workgroup
// reads together from every page.
int heads_per_group(int hkv, int max_waves) {
  for (int d = max_waves; d > 1; --d)
    if (hkv % d == 0) return d;
  return 1;
}

// Workgroups: one wave per kv head of a group of hgs, times step phases up
// to max_waves(d) waves (8; 4 at D = 256); as many workgroups as fill the
// device (blocks_per_cu per CU), but none with fewer than min_steps 32-token
// steps per wave at the largest context the page table allows.  Partial
// slots: one per (workgroup, sequence piece), at most grid + batch * kv-head
// groups, each holding `cols` (query token, head) rows per kv head.
Plan plan_for(int hgs, int32_t batch, int32_t hkv, int32_t d, int32_t p, int32_t maxp, int num_cus, int cols,
              int min_steps) {
  Plan pl;
  const int max_waves = pda::max_waves(d);
  pl.hgs = hgs;
  pl.min_steps = min_steps;
  const int phases = max_waves / pl.hgs;
  pl.waves = pl.hgs * phases;
  const int64_t ngroups = hkv / pl.hgs;
  const int64_t max_ctx = static_cast<int64_t>(maxp) * p;
  const int64_t steps_max = static_cast<int64_t>(batch) * ngroups * ((max_ctx + pda::kStep - 1) / pda::kStep);
  const int64_t per_block = static_cast<int64_t>(min_steps) * phases;
  int64_t blocks = (steps_max + per_block - 1) / per_block;
  const int64_t target = static_cast<int64_t>(num_cus) * blocks_per_cu();
  if (blocks > target) blocks = target;
  if (blocks < 1) blocks = 1;
  pl.grid = static_cast<int>(blocks);
  pl.slots = static_cast<int64_t>(pl.grid) + static_cast<int64_t>(batch) * ngroups;
  const int64_t rows = pl.slots * pl.hgs * cols;
  pl.off_acc = 0;
  pl.off_ml = align256(rows * d * 4);
  pl.off_pref = pl.off_ml + align256(rows * 2 * 4);
  // steps prefix [batch + 1], then the split list [grid] (see the kernels)
  pl.bytes = pl.off_pref + align256((static_cast<int64_t>(batch) + 1 + pl.grid) * 4);
  return pl;
}

// The fixed split of a latency-bound call with the kv-head grouping and
// step count of `base`: every (sequence, kv-head group) is cut into the same
// number of chunks of whole 32-token steps, as many as the stream-K plan
// would give it at the page table's largest context (but at least 2 and
// within the device's workgroups), so each workgroup knows its piece from
// its index.  Where the stream-K plan takes a single workgroup, every pair is
// one chunk: whole sequences, one workgroup each, nothing to merge.  Returns
// a plan with grid 0 where it does not apply: more pairs than half the
// device's workgroups (the stream-K split balances those better).  One
// partial slot per workgroup.
Plan plan_fixed(const Plan& base, int32_t batch, int32_t hkv, int32_t d, int32_t p, int32_t maxp, int num_cus,
                int cols) {
  Plan pl = base;
  pl.grid = 0;
  const int phases = pl.waves / pl.hgs;
  const int64_t seqs = static_cast<int64_t>(batch) * (hkv / pl.hgs);
  const int64_t target = static_cast<int64_t>(num_cus) * blocks_per_cu();
  const int64_t max_ctx = static_cast<int64_t>(maxp) * p;
  const int64_t steps_seq = (max_ctx + pda::kStep - 1) / pda::kStep;
  const int64_t per_block = static_cast<int64_t>(pl.min_steps) * phases;
  if (base.grid < 1 || 2 * seqs > target) return pl;
  int64_t chunks = 1;
  if (base.grid > 1) {
    chunks = std::min((steps_seq + per_block - 1) / per_block, target / seqs);
    chunks = std::max<int64_t>(chunks, 1);
  }
  const int64_t chunk_steps = (steps_seq + chunks - 1) / chunks;
  chunks = (steps_seq + chunk_steps - 1) / chunk_steps;  // no chunk wholly past the largest context
  if (base.grid > 1 && chunks < 2) return pl;
  pl.grid = static_cast<int>(seqs * chunks);
  pl.chunks = static_cast<int>(chunks);
  pl.chunk_steps = static_cast<int>(chunk_steps);
  pl.slots = pl.grid;
  const int64_t rows = pl.slots * pl.hgs * cols;
  pl.off_acc = 0;
  pl.off_ml = align256(rows * d * 4);
  pl.off_pref = pl.off_ml + align256(rows * 2 * 4);
  pl.bytes = pl.off_pref + align256((static_cast<int64_t>(batch) + 1 + pl.grid) * 4);
  return pl;
}

// The plan of a call.  The default reads all kv heads of a group of up to 8
// together (the faster access order for long streams) and merges split
// sequences in a separate kernel.  With PDA_OPT_FUSED_MERGE = 1, a grid of
// several workgroups with little partial data per sequence merges inside
// the attention kernel instead: with the largest kv-head group for which
// the most partial data one sequence can have, grid x hgs x cols x d fp32,
// fits pda::kFusedMergeBytes (a single request then takes one kv head per
// workgroup); a latency-bound call with the fixed split keeps it, its
// sequences merged by the last of their chunks (1 x 4096 tokens, 32:8
// heads: 14.0 us per call against 11.7 us with the merge kernel).  On
// MI355X the in-kernel hand-off (write-through stores, their
// acknowledgement, the arrival atomic, coherent reloads) costs more than
// the merge kernel's launch, so the option is off by default.
// Calls whose K and V (bounded by the page table) fit in this many bytes are
// latency-bound: they take the small-call rules of make_plan.
constexpr int64_t kSmallCallBytes = int64_t{128} << 20;
// Most pieces a small call cuts one (sequence, kv-head group) into.
constexpr int64_t kSmallCallPieces = 32;
constexpr int kDefaultMinSteps = 2;

Plan make_plan(int32_t batch, int32_t hkv, int32_t d, int32_t p, int32_t maxp, int num_cus, int cols) {
  const int cap = kv_group_cap();
  const int ms_opt = min_steps_option();
  // A split piece leaves a partial of cols x head_dim fp32 per kv head it
  // covers; with more than 8 columns (several query tokens) those writes
  // cost more than the longer token rows save, so at most 4 kv heads go
  // together (multiq: 191.4 -> 188.3 us per call; long70b and ragged, at 8
  // columns or fewer, run slower with 4).
  const int dflt_most = cols > 8 ? std::min(4, pda::max_waves(d)) : pda::max_waves(d);
  const int most = cap > 0 && cap < pda::max_waves(d) ? cap : dflt_most;
  Plan dflt = plan_for(heads_per_group(hkv, most), batch, hkv, d, p, maxp, num_cus, cols,
                       ms_opt > 0 ? ms_opt : kDefaultMinSteps);
  // Small calls (each 32-token step's K and V is a few KB; the whole call
  // is a chain of latencies):
  //  - a plan that splits the work but leaves CUs idle gives each wave one
  //    step instead of two, doubling the workgroups (graph replay of 20
  //    calls over cold K/V: 1 x 1024 tokens 15.1 -> 12.5 us, 4 x 1024
  //    15.9 -> 13.6, 8 x 512 15.7 -> 13.8);
  //  - fewer kv heads per workgroup when a sequence's heads would be cut
  //    into more than kSmallCallPieces pieces: the same workgroups then take
  //    longer runs of fewer heads, so less partial data and a lighter merge
  //    (1 x 4096 tokens, 32:8 heads, 15.6 -> 14.4 us with 2 heads per
  //    workgroup; 1 x 16384 25.1 -> 21.9 with 1; 1 x 8192, 64:8 heads,
  //    20.7 -> 16.8 with 1).  Large calls keep 8 heads, whose 2 KB token
  //    rows stream faster (long70b: 319.8 us per call with 8, 321.2 with 4,
  //    329.6 with 2, 351.8 with 1).
  //  - the fixed split (plan_fixed) unless PDA_OPT_FIXED_SPLIT is 0: the
  //    first K/V loads leave ~2 us earlier and the merge needs no prefix
  //    (1 x 4096 tokens, 32:8 heads, cold K/V: attention kernel 14.8 ->
  //    11.4 us by events, 16.7 -> 11.9 us per call replayed from a graph).
  const int64_t kv_bytes = static_cast<int64_t>(batch) * maxp * p * hkv * d * 4;
  const bool small = kv_bytes <= kSmallCallBytes;
  if (small) {
    if (ms_opt == 0 && dflt.grid > 1 && dflt.grid < static_cast<int64_t>(num_cus) * blocks_per_cu())
      dflt = plan_for(dflt.hgs, batch, hkv, d, p, maxp, num_cus, cols, 1);
    if (cap == 0) {
      for (int h = dflt.hgs; h >= 1; --h) {
        if (hkv % h) continue;
        if (h == 1 || static_cast<int64_t>(dflt.grid) * h <= kSmallCallPieces * batch * hkv) {
          if (h != dflt.hgs) dflt = plan_for(h, batch, hkv, d, p, maxp, num_cus, cols, dflt.min_steps);
          break;
        }
      }
    }
  }
  // (the vector-ALU variant, a measurement aid, keeps the merge kernel)
  if (dflt.grid == 1 || !fused_merge() || compute_path() != 0) {
    if (small && fixed_split() && compute_path() == 0) {
      const Plan f = plan_fixed(dflt, batch, hkv, d, p, maxp, num_cus, cols);
      if (f.grid > 0) return f;
    }
    return dflt;
  }
  // a latency-bound call keeps the fixed split, merged in the kernel
  if (small && fixed_split()) {
    Plan f = plan_fixed(dflt, batch, hkv, d, p, maxp, num_cus, cols);
    if (f.grid > 1 && f.chunks > 1 && f.grid <= pda::kMaxFusedGrid) {
      f.fused = true;
      return f;
    }
  }
  if (fused_merge() == 2) {  // every plan that has something to merge (tests)
    Plan c = dflt;
    c.fused = c.grid <= pda::kMaxFusedGrid && c.bytes < (int64_t{1} << 31);
    return c;
  }
  for (int h = dflt.hgs; h >= 1; --h) {
    if (hkv % h) continue;
    Plan c = plan_for(h, batch, hkv, d, p, maxp, num_cus, cols, dflt.min_steps);
    const int64_t most_bytes = static_cast<int64_t>(c.grid) * h * cols * d * 4;
    if (c.grid > 1 && c.grid <= pda::kMaxFusedGrid && most_bytes <= pda::kFusedMergeBytes &&
        c.bytes < (int64_t{1} << 31)) {
      c.fused = true;
      return c;
    }
  }
  return dflt;
}

// Workspace that any call of this shape may need: the largest plan over
// every kv-head group size and step count make_plan can pick, at 16 columns
// per kv head.
int64_t reserve_bytes(int32_t batch, int32_t hkv, int32_t d, int32_t p, int32_t maxp, int num_cus) {
  const int ms_opt = min_steps_option();
  int64_t most = 0;
  for (int ms : {ms_opt > 0 ? ms_opt : kDefaultMinSteps, ms_opt > 0 ? ms_opt : 1})
    for (int h = 1; h <= pda::max_waves(d); ++h)
      if (hkv % h == 0) {
        const Plan pl = plan_for(h, batch, hkv, d, p, maxp, num_cus, pda::kMaxCols, ms);
        most = std::max(most, pl.bytes);
        most = std::max(most, plan_fixed(pl, batch, hkv, d, p, maxp, num_cus, pda::kMaxCols).bytes);
      }
  return most;
}

int device_cus(int dev, int* cus) {
  static std::mutex mu;
  static std::map<int, int> cache;
  std::lock_guard<std::mutex> lock(mu);
  auto it = cache.find(dev);
  if (it != cache.end()) {
    *cus = it->second;
    return PDA_OK;
  }
  int n = 0;
  hipError_t e = hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev);
  if (e != hipSuccess) return hip_fail(e, "hipDeviceGetAttribute(multiprocessor count)");
  cache[dev] = n;
  *cus = n;
  return PDA_OK;
}

// ---------------------------------------------------------------- workspaces
// Per (device, stream): one buffer for split partials and the steps prefix.
struct Workspace {
  void* ptr = nullptr;
  int64_t bytes = 0;
  int32_t* cnt = nullptr;  // arrival counters of the fused merge, zero between calls
};
std::mutex g_ws_mu;
std::map<std::pair<int, hipStream_t>, Workspace> g_ws;

int workspace_for(int dev, hipStream_t st, int64_t need, void** out) {
  std::lock_guard<std::mutex> lock(g_ws_mu);
  Workspace& ws = g_ws[{dev, st}];
  if (ws.bytes >= need) {
    *out = ws.ptr;
    return PDA_OK;
  }
  hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
  hipError_t e = hipStreamIsCapturing(st, &cap);
  if (e != hipSuccess) return hip_fail(e, "hipStreamIsCapturing");
  if (cap != hipStreamCaptureStatusNone)
    return fail(PDA_ERR_HIP, "workspace must grow to %lld bytes while the stream is being captured; "
                "call pda_workspace_reserve before capture", static_cast<long long>(need));
  if (ws.ptr) {
    e = hipStreamSynchronize(st);  // in-flight calls may still use the old buffer
    if (e != hipSuccess) return hip_fail(e, "hipStreamSynchronize");
    if ((e = hipFree(ws.ptr)) != hipSuccess) return hip_fail(e, "hipFree");
    ws.ptr = nullptr;
    ws.bytes = 0;
  }
  const int64_t grow = need + need / 4;
  if ((e = hipMalloc(&ws.ptr, static_cast<size_t>(grow))) != hipSuccess) {
    ws.ptr = nullptr;
    return hip_fail(e, "hipMalloc(workspace)");
  }
  ws.bytes = grow;
  *out = ws.ptr;
  return PDA_OK;
}

// The fused merge's arrival counters of (device, stream): a buffer of their
// own (the GEMV calls share the workspace), cleared once when allocated;
// every call leaves them at zero.
int counters_for(int dev, hipStream_t st, int32_t** out) {
  std::lock_guard<std::mutex> lock(g_ws_mu);
  Workspace& ws = g_ws[{dev, st}];
  if (!ws.cnt) {
    hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
    hipError_t e = hipStreamIsCapturing(st, &cap);
    if (e != hipSuccess) return hip_fail(e, "hipStreamIsCapturing");
    if (cap != hipStreamCaptureStatusNone)
      return fail(PDA_ERR_HIP, "the merge counters must be allocated while the stream is being captured; "
                  "call pda_workspace_reserve before capture");
    void* p = nullptr;
    const size_t bytes = static_cast<size_t>(pda::kMaxFusedGrid) * sizeof(int32_t);
    if ((e = hipMalloc(&p, bytes)) != hipSuccess) return hip_fail(e, "hipMalloc(merge counters)");
    if ((e = hipMemsetAsync(p, 0, bytes, st)) != hipSuccess) {
      (void)hipFree(p);
      return hip_fail(e, "hipMemsetAsync(merge counters)");
    }
    ws.cnt = static_cast<int32_t*>(p);
  }
  *out = ws.cnt;
  return PDA_OK;
}

// ---------------------------------------------------------------- profiling
// Events around the two kernels of a call: kind 0 is attention (split,
// merge), kind 1 the prelude (GEMV, epilogue), kind 2 o_proj (GEMV, epilogue).
struct Rec {
  hipEvent_t a, b, c;
  int kind;
};
std::mutex g_prof_mu;
bool g_prof_on = false;
std::vector<Rec> g_prof_recs;
std::vector<hipEvent_t> g_prof_pool;

hipEvent_t prof_event() {
  if (!g_prof_pool.empty()) {
    hipEvent_t e = g_prof_pool.back();
    g_prof_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

// A record with three events when profiling is on, else one with none.
Rec prof_begin(int kind) {
  std::lock_guard<std::mutex> lock(g_prof_mu);
  if (!g_prof_on) return Rec{nullptr, nullptr, nullptr, kind};
  Rec r{prof_event(), prof_event(), prof_event(), kind};
  if (!r.a || !r.b || !r.c) return Rec{nullptr, nullptr, nullptr, kind};
  return r;
}

void prof_push(const Rec& r) {
  std::lock_guard<std::mutex> lock(g_prof_mu);
  g_prof_recs.push_back(r);
}

// Sum the two intervals of every record of `kind`, release them.
int prof_read(int kind, double* first_ms, double* second_ms, int64_t* calls) {
  std::lock_guard<std::mutex> lock(g_prof_mu);
  double s = 0, m = 0;
  int64_t n = 0;
  int rc = PDA_OK;
  std::vector<Rec> keep;
  for (const Rec& r : g_prof_recs) {
    if (r.kind != kind) {
      keep.push_back(r);
      continue;
    }
    float t1 = 0, t2 = 0;
    hipError_t e = hipEventSynchronize(r.c);
    if (e == hipSuccess) e = hipEventElapsedTime(&t1, r.a, r.b);
    if (e == hipSuccess) e = hipEventElapsedTime(&t2, r.b, r.c);
    if (e != hipSuccess) rc = hip_fail(e, "reading profile events");
    s += t1;
    m += t2;
    ++n;
    g_prof_pool.push_back(r.a);
    g_prof_pool.push_back(r.b);
    g_prof_pool.push_back(r.c);
  }
  g_prof_recs.swap(keep);
  *first_ms = s;
  *second_ms = m;
  *calls = n;
  return rc;
}

// ---------------------------------------------------------------- validation
// Host-side check of the device page tables and lengths (debugging aid):
// synchronises the stream and copies both to the host.
int validate_paging(const int32_t* block_table, const int32_t* context_lens, int32_t batch, int32_t maxp,
                    int32_t page_size, int32_t num_pages, hipStream_t st) {
  std::vector<int32_t> lens(batch), bt(static_cast<size_t>(batch) * maxp);
  hipError_t e = hipMemcpyAsync(lens.data(), context_lens, lens.size() * 4, hipMemcpyDeviceToHost, st);
  if (e == hipSuccess)
    e = hipMemcpyAsync(bt.data(), block_table, bt.size() * 4, hipMemcpyDeviceToHost, st);
  if (e == hipSuccess) e = hipStreamSynchronize(st);
  if (e != hipSuccess) return hip_fail(e, "reading block_table / context_lens for validation");
  const int64_t max_ctx = static_cast<int64_t>(maxp) * page_size;
  for (int32_t b = 0; b < batch; ++b) {
    if (lens[b] < 0 || lens[b] > max_ctx)
      return fail(PDA_ERR_SHAPE, "context_lens[%d] = %d outside [0, %lld]", b, lens[b],
                  static_cast<long long>(max_ctx));
    const int32_t pages = (lens[b] + page_size - 1) / page_size;
    for (int32_t j = 0; j < pages; ++j) {
      const int32_t id = bt[static_cast<size_t>(b) * maxp + j];
      if (id < 0 || id >= num_pages)
        return fail(PDA_ERR_SHAPE, "block_table[%d][%d] = %d outside [0, %d)", b, j, id, num_pages);
    }
  }
  return PDA_OK;
}

// PDA_DEBUG_VALIDATE=1: check the paging inputs before every attention or
// append call (skipped while the stream is being captured).
bool debug_validate() {
  static const bool on = env_int("PDA_DEBUG_VALIDATE", 0, 0, 1) == 1;
  return on;
}

int maybe_validate(const int32_t* block_table, const int32_t* context_lens, int32_t batch, int32_t maxp,
                   int32_t page_size, int32_t num_pages, hipStream_t st) {
  if (!debug_validate()) return PDA_OK;
  hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
  if (hipStreamIsCapturing(st, &cap) != hipSuccess || cap != hipStreamCaptureStatusNone) return PDA_OK;
  return validate_paging(block_table, context_lens, batch, maxp, page_size, num_pages, st);
}


// ---------------------------------------------------------------- descriptors
const char* dtype_name(int32_t dt) {
  switch (dt) {
    case PDA_DTYPE_BF16: return "bf16";
    case PDA_DTYPE_F16: return "fp16";
    case PDA_DTYPE_F32: return "fp32";
    case PDA_DTYPE_I32: return "int32";
    case PDA_DTYPE_I64: return "int64";
    default: return "unknown";
  }
}

// Rank and extents of one descriptor (not NULL).
int check_rank(const pda_tensor& t, const char* name, int32_t ndim) {
  if (t.ndim != ndim) return fail(PDA_ERR_SHAPE, "%s: %d dimensions, expected %d", name, t.ndim, ndim);
  for (int i = 0; i < ndim; ++i)
    if (t.shape[i] < 0 || t.shape[i] > INT32_MAX)
      return fail(PDA_ERR_SHAPE, "%s: extent %lld of dimension %d out of range", name,
                  static_cast<long long>(t.shape[i]), i);
  return PDA_OK;
}

bool desc_empty(const pda_tensor& t) {
  for (int i = 0; i < t.ndim; ++i)
    if (t.shape[i] == 0) return true;
  return false;
}

// Dense row-major strides (extent-1 dimensions and empty tensors excepted).
int check_dense(const pda_tensor& t, const char* name) {
  if (desc_empty(t)) return PDA_OK;
  int64_t want = 1;
  for (int i = t.ndim - 1; i >= 0; --i) {
    if (t.shape[i] != 1 && t.stride[i] != want)
      return fail(PDA_ERR_LAYOUT, "%s: stride %lld in dimension %d, a dense row-major tensor has %lld", name,
                  static_cast<long long>(t.stride[i]), i, static_cast<long long>(want));
    if (want > (int64_t{1} << 50) / (t.shape[i] > 0 ? t.shape[i] : 1))
      return fail(PDA_ERR_SHAPE, "%s: too many elements", name);
    want *= t.shape[i];
  }
  return PDA_OK;
}

// ---------------------------------------------------------------- prelude
bool misaligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) != 0; }

int check_prelude(const pda_prelude_dims* dm) {
  if (!dm) return fail(PDA_ERR_NULL, "dims is NULL");
  const pda_prelude_dims& d = *dm;
  if (d.batch < 0) return fail(PDA_ERR_SHAPE, "batch must be >= 0 (got %d)", d.batch);
  if (d.batch > pda::kMaxGemvBatch)
    return fail(PDA_ERR_UNSUPPORTED, "prelude batch %d exceeds %d", d.batch, pda::kMaxGemvBatch);
  if (d.hidden <= 0 || d.num_q_heads <= 0 || d.num_kv_heads <= 0)
    return fail(PDA_ERR_SHAPE, "hidden and head counts must be positive");
  if (d.hidden % pda::kTileK || d.hidden > 65536)
    return fail(PDA_ERR_UNSUPPORTED, "hidden %d (supported: multiples of 32 up to 65536)", d.hidden);
  if (d.num_q_heads % d.num_kv_heads)
    return fail(PDA_ERR_SHAPE, "num_q_heads %d is not a multiple of num_kv_heads %d", d.num_q_heads,
                d.num_kv_heads);
  if (d.head_dim != 64 && d.head_dim != 128 && d.head_dim != 256)
    return fail(PDA_ERR_UNSUPPORTED, "head_dim %d (supported: 64, 128, 256)", d.head_dim);
  if (d.batch > pda::kMaxGemvBatchAnyRows &&
      (static_cast<int64_t>(d.num_q_heads + 2 * d.num_kv_heads) * d.head_dim) % 128)
    return fail(PDA_ERR_UNSUPPORTED, "prelude batch %d above %d needs (num_q_heads + 2 num_kv_heads) * head_dim "
                "a multiple of 128", d.batch, pda::kMaxGemvBatchAnyRows);
  if (d.num_kv_heads > PDA_MAX_KV_HEADS || d.num_q_heads > 8 * PDA_MAX_KV_HEADS)
    return fail(PDA_ERR_UNSUPPORTED, "too many heads (q %d, kv %d)", d.num_q_heads, d.num_kv_heads);
  if (d.rotary_dim < 0 || d.rotary_dim > d.head_dim || (d.rotary_dim & 1))
    return fail(PDA_ERR_SHAPE, "rotary_dim %d (0, or even up to head_dim %d)", d.rotary_dim, d.head_dim);
  if (d.interleaved != 0 && d.interleaved != 1) return fail(PDA_ERR_SHAPE, "interleaved must be 0 or 1");
  if (!std::isfinite(d.rope_theta) || !(d.rope_theta > 0.f))
    return fail(PDA_ERR_SCALE, "rope_theta must be finite and > 0");
  if (!std::isfinite(d.eps) || d.eps < 0.f) return fail(PDA_ERR_SCALE, "eps must be finite and >= 0");
  return PDA_OK;
}

int64_t prelude_rows(const pda_prelude_dims& d) {
  return static_cast<int64_t>(d.num_q_heads + 2 * d.num_kv_heads) * d.head_dim;
}

// The GEMV plan of a prelude on this device's compute units.
pda::GemvPlan prelude_plan(const pda_prelude_dims& d, int cus) {
  return pda::plan_gemv(d.batch, static_cast<int>(prelude_rows(d)), d.hidden, cus);
}

int64_t prelude_ws_bytes(const pda_prelude_dims& d, int cus) {
  return align256(pda::gemv_partial_floats(prelude_plan(d, cus), d.batch, static_cast<int>(prelude_rows(d))) * 4);
}

// o_proj workspace: GEMV partials, then z [batch, hidden] and the chunk sums.
int64_t oproj_z_offset(const pda::GemvPlan& plan, int batch, int hidden) {
  return align256(pda::gemv_partial_floats(plan, batch, hidden) * 4);
}

int64_t oproj_ws_bytes(const pda::GemvPlan& plan, int batch, int hidden) {
  return oproj_z_offset(plan, batch, hidden) +
         align256((static_cast<int64_t>(batch) * hidden + static_cast<int64_t>(batch) * pda::oproj_chunks(hidden)) * 4);
}

// Shared by both prelude entry points once their own arguments are checked.
int run_prelude(const void* x, const void* w_packed, const void* bias, const void* q_norm, const void* k_norm,
                const int32_t* context_lens, void* q_out, pda::PreludeArgs ep, const pda_prelude_dims& d,
                void* stream) {
  if (!x || !w_packed || !context_lens || !q_out) return fail(PDA_ERR_NULL, "a tensor pointer is NULL");
  if ((q_norm == nullptr) != (k_norm == nullptr))
    return fail(PDA_ERR_NULL, "q_norm and k_norm must both be given or both be NULL");
  if (misaligned(x, 16) || misaligned(w_packed, 16) || misaligned(q_out, 16))
    return fail(PDA_ERR_ALIGN, "x, w_packed and the outputs must be 16-byte aligned");
  if (misaligned(bias, 2) || misaligned(q_norm, 2) || misaligned(k_norm, 2) || misaligned(context_lens, 4))
    return fail(PDA_ERR_ALIGN, "bias / norm weights must be 2-byte and context_lens 4-byte aligned");
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  int cus = 0;
  int rc = device_cus(dev, &cus);
  if (rc) return rc;
  hipStream_t st = static_cast<hipStream_t>(stream);
  void* ws = nullptr;
  if ((rc = workspace_for(dev, st, prelude_ws_bytes(d, cus), &ws))) return rc;
  pda::GemvArgs g;
  g.x = static_cast<const uint16_t*>(x);
  g.wp = static_cast<const uint16_t*>(w_packed);
  g.part = static_cast<float*>(ws);
  g.batch = d.batch;
  g.n = static_cast<int>(prelude_rows(d));
  g.k = d.hidden;
  g.plan = prelude_plan(d, cus);
  const Rec rec = prof_begin(1);
  const bool prof = rec.a != nullptr;
  if (prof && (e = hipEventRecord(rec.a, st)) != hipSuccess) return hip_fail(e, "hipEventRecord");
  if ((e = pda::launch_gemv(g, st)) != hipSuccess) return hip_fail(e, "GEMV kernel launch");
  if (prof && (e = hipEventRecord(rec.b, st)) != hipSuccess) return hip_fail(e, "hipEventRecord");
  ep.part = g.part;
  ep.plan = g.plan;
  ep.bias = static_cast<const uint16_t*>(bias);
  ep.q_norm = static_cast<const uint16_t*>(q_norm);
  ep.k_norm = static_cast<const uint16_t*>(k_norm);
  ep.lens = context_lens;
  ep.q_out = static_cast<uint16_t*>(q_out);
  ep.batch = d.batch;
  ep.hq = d.num_q_heads;
  ep.hkv = d.num_kv_heads;
  ep.d = d.head_dim;
  ep.rotary_dim = d.rotary_dim;
  ep.interleaved = d.interleaved;
  {
    const double log2_theta = std::log2(static_cast<double>(d.rope_theta));
    for (int k = 0; k < 8; ++k)
      ep.freq_pow2[k] = d.rotary_dim > 0 ? std::exp2(-(2.0 * (1 << k) / d.rotary_dim) * log2_theta) : 0.0;
  }
  ep.eps = d.eps;
  if ((e = pda::launch_prelude_epilogue(ep, st)) != hipSuccess) return hip_fail(e, "prelude epilogue launch");
  if (prof) {
    if ((e = hipEventRecord(rec.c, st)) != hipSuccess) return hip_fail(e, "hipEventRecord");
    prof_push(rec);
  }
  return PDA_OK;
}

// The attention entry points: argument checks, plan, workspace, launches.
// noalloc: the workspace is the library's fixed per-device scratch (no
// allocation, no paging validation, no profiling events) instead of the
// (device, stream) workspace, and shapes whose plan needs more than it
// holds are rejected.
int attention_call(const void* q, const void* k_cache, const void* v_cache, const int32_t* block_table,
                   const int32_t* context_lens, void* out, int32_t batch, int32_t num_q_heads,
                   int32_t num_kv_heads, int32_t head_dim, int32_t page_size, int32_t num_pages,
                   int32_t max_pages_per_seq, int32_t num_queries, int32_t window, float scale, void* stream,
                   bool noalloc) {
  g_err.clear();
  int rc = check_attention(batch, num_q_heads, num_kv_heads, head_dim, page_size, max_pages_per_seq);
  if (rc) return rc;
  if (num_pages <= 0) return fail(PDA_ERR_SHAPE, "num_pages must be positive (got %d)", num_pages);
  if (num_queries < 1) return fail(PDA_ERR_SHAPE, "num_queries must be >= 1 (got %d)", num_queries);
  if (window < 0) return fail(PDA_ERR_SHAPE, "window must be >= 0 (got %d)", window);
  if (num_queries > pda::kMaxCols || num_queries * (num_q_heads / num_kv_heads) > pda::kMaxCols)
    return fail(PDA_ERR_UNSUPPORTED, "num_queries %d x query group %d exceeds %d", num_queries,
                num_q_heads / num_kv_heads, pda::kMaxCols);
  if (!std::isfinite(scale)) return fail(PDA_ERR_SCALE, "scale is not finite");
  const int cols = num_queries * (num_q_heads / num_kv_heads);
  int valu_cols = 0;
  if ((rc = check_compute_path(head_dim, page_size, cols, batch, &valu_cols))) return rc;
  if (batch == 0) return PDA_OK;
  if (!q || !k_cache || !v_cache || !block_table || !context_lens || !out)
    return fail(PDA_ERR_NULL, "a tensor pointer is NULL");
  auto misaligned = [](const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) != 0; };
  if (misaligned(q, 16) || misaligned(k_cache, 16) || misaligned(v_cache, 16) || misaligned(out, 16))
    return fail(PDA_ERR_ALIGN, "q, k_cache, v_cache and out must be 16-byte aligned");
  if (misaligned(block_table, 4) || misaligned(context_lens, 4))
    return fail(PDA_ERR_ALIGN, "block_table and context_lens must be 4-byte aligned");
  if (!noalloc && (rc = maybe_validate(block_table, context_lens, batch, max_pages_per_seq, page_size,
                                       num_pages, static_cast<hipStream_t>(stream))))
    return rc;

  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  int cus = 0;
  if ((rc = device_cus(dev, &cus))) return rc;
  const Plan pl = make_plan(batch, num_kv_heads, head_dim, page_size, max_pages_per_seq, cus, cols);
  if (pda::attn_lds_bytes(head_dim, batch, pl.waves, valu_cols > 0) > static_cast<size_t>(pda::kMaxLdsBytes))
    return fail(PDA_ERR_UNSUPPORTED, "batch %d needs more LDS than a workgroup has", batch);
  hipStream_t st = static_cast<hipStream_t>(stream);
  void* ws = nullptr;
  int32_t* cnt = nullptr;
  if (noalloc) {
    // the partials from the start of the scratch, the merge counters at its end
    const int64_t counter_bytes = static_cast<int64_t>(pda::kMaxFusedGrid) * 4;
    if (pl.bytes > PDA_NOALLOC_SCRATCH_BYTES - counter_bytes)
      return fail(PDA_ERR_UNSUPPORTED,
                  "this shape needs %lld bytes of workspace; the no-allocation entry point holds %lld",
                  static_cast<long long>(pl.bytes), static_cast<long long>(PDA_NOALLOC_SCRATCH_BYTES - counter_bytes));
    if ((e = pda::noalloc_scratch(dev, &ws)) != hipSuccess) return hip_fail(e, "hipGetSymbolAddress(scratch)");
    cnt = reinterpret_cast<int32_t*>(static_cast<char*>(ws) + PDA_NOALLOC_SCRATCH_BYTES - counter_bytes);
  } else {
    if ((rc = workspace_for(dev, st, pl.bytes, &ws))) return rc;
    if (pl.fused && (rc = counters_for(dev, st, &cnt))) return rc;
  }

  pda::LaunchArgs a;
  a.q = static_cast<const uint16_t*>(q);
  a.k = static_cast<const uint16_t*>(k_cache);
  a.v = static_cast<const uint16_t*>(v_cache);
  a.bt = block_table;
  a.lens = context_lens;
  a.out = static_cast<uint16_t*>(out);
  a.ws_acc = reinterpret_cast<float*>(static_cast<char*>(ws) + pl.off_acc);
  a.ws_ml = reinterpret_cast<float*>(static_cast<char*>(ws) + pl.off_ml);
  a.ws_pref = reinterpret_cast<int32_t*>(static_cast<char*>(ws) + pl.off_pref);
  a.batch = batch;
  a.hq = num_q_heads;
  a.hkv = num_kv_heads;
  a.group = num_q_heads / num_kv_heads;
  a.head_dim = head_dim;
  a.page_shift = log2i(page_size);
  a.num_pages = num_pages;
  a.maxp = max_pages_per_seq;
  a.grid = pl.grid;
  a.waves = pl.waves;
  a.hgs = pl.hgs;
  a.min_steps = pl.min_steps;
  a.scale = scale;
  a.nq = num_queries;
  a.window = window;
  a.valu_cols = valu_cols;
  a.ws_cnt = cnt;
  a.fused = pl.fused;
  a.chunks = pl.chunks;
  a.chunk_steps = pl.chunk_steps;
  // the first-piece stash of stream-K plans, where the LDS holds it
  a.stash = pl.chunks == 0 && !pl.fused && pl.grid > 1 && valu_cols == 0 &&
            pda::attn_stash_lds_bytes(head_dim, batch, pl.waves, pl.hgs, cols, valu_cols > 0) <=
                static_cast<size_t>(pda::kMaxLdsBytes);

  const Rec rec = noalloc ? Rec{nullptr, nullptr, nullptr, 0} : prof_begin(0);
  const bool prof = rec.a != nullptr;
  if (prof && (e = hipEventRecord(rec.a, st)) != hipSuccess) return hip_fail(e, "hipEventRecord");
  if ((e = pda::launch_attn_kernel(a, st)) != hipSuccess) return hip_fail(e, "attention kernel launch");
  if (prof && (e = hipEventRecord(rec.b, st)) != hipSuccess) return hip_fail(e, "hipEventRecord");
  // with one workgroup, or one fixed-split chunk per sequence, every piece
  // is a whole sequence: nothing to merge; a fused plan merged in the
  // attention kernel
  if (pl.grid > 1 && !pl.fused && pl.chunks != 1 && (e = pda::launch_merge_kernel(a, st)) != hipSuccess)
    return hip_fail(e, "merge kernel launch");
  if (prof) {
    if ((e = hipEventRecord(rec.c, st)) != hipSuccess) return hip_fail(e, "hipEventRecord");
    prof_push(rec);
  }
  return PDA_OK;
}

}  // namespace

extern "C" {

const char* pda_last_error(void) { return g_err.c_str(); }

int32_t pda_version(void) { return PDA_VERSION; }

int pda_plan(int32_t batch, int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
             int32_t page_size, int32_t max_pages_per_seq, int32_t num_cus, int32_t* grid_blocks,
             int32_t* waves, int64_t* workspace_bytes) {
  g_err.clear();
  if (!grid_blocks || !waves || !workspace_bytes) return fail(PDA_ERR_NULL, "pda_plan: NULL output pointer");
  int rc = check_attention(batch, num_q_heads, num_kv_heads, head_dim, page_size, max_pages_per_seq);
  if (rc) return rc;
  if (num_cus <= 0) return fail(PDA_ERR_SHAPE, "num_cus must be positive");
  Plan pl = make_plan(batch, num_kv_heads, head_dim, page_size, max_pages_per_seq, num_cus,
                      num_q_heads / num_kv_heads);
  *grid_blocks = batch ? pl.grid : 0;
  *waves = batch ? pl.grid * pl.waves : 0;
  *workspace_bytes =
      batch ? reserve_bytes(batch, num_kv_heads, head_dim, page_size, max_pages_per_seq, num_cus) : 0;
  return PDA_OK;
}

int pda_workspace_reserve(int32_t batch, int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
                          int32_t page_size, int32_t max_pages_per_seq, void* stream) {
  g_err.clear();
  int rc = check_attention(batch, num_q_heads, num_kv_heads, head_dim, page_size, max_pages_per_seq);
  if (rc) return rc;
  if (batch == 0) return PDA_OK;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  int cus = 0;
  if ((rc = device_cus(dev, &cus))) return rc;
  // sized for the most (query token, head) columns, so any num_queries fits
  void* ptr = nullptr;
  const int64_t need = reserve_bytes(batch, num_kv_heads, head_dim, page_size, max_pages_per_seq, cus);
  if ((rc = workspace_for(dev, static_cast<hipStream_t>(stream), need, &ptr))) return rc;
  int32_t* cnt = nullptr;
  return counters_for(dev, static_cast<hipStream_t>(stream), &cnt);
}

int pda_release_workspaces(void) {
  g_err.clear();
  std::lock_guard<std::mutex> lock(g_ws_mu);
  int rc = PDA_OK;
  for (auto& kv : g_ws) {
    if (!kv.second.ptr && !kv.second.cnt) continue;
    int cur = 0;
    hipError_t e = hipGetDevice(&cur);
    if (e == hipSuccess) e = hipSetDevice(kv.first.first);
    if (e == hipSuccess) e = hipStreamSynchronize(kv.first.second);
    if (e == hipSuccess && kv.second.ptr) e = hipFree(kv.second.ptr);
    if (e == hipSuccess && kv.second.cnt) e = hipFree(kv.second.cnt);
    const hipError_t back = hipSetDevice(cur);
    if (e == hipSuccess) e = back;
    if (e != hipSuccess) rc = hip_fail(e, "releasing a workspace");
  }
  g_ws.clear();
  return rc;
}

int pda_set_option(int32_t option, int32_t value) {
  g_err.clear();
  switch (option) {
    case PDA_OPT_BLOCKS_PER_CU:
      if (value < 1 || value > kMaxBlocksPerCu)
        return fail(PDA_ERR_SHAPE, "blocks per CU must be in [1, %d]", kMaxBlocksPerCu);
      g_blocks_per_cu.store(value);
      return PDA_OK;
    case PDA_OPT_MIN_STEPS:
      if (value < 0) return fail(PDA_ERR_SHAPE, "min steps per wave must be >= 0 (0 = the planner's choice)");
      g_min_steps.store(value);
      return PDA_OK;
    case PDA_OPT_COMPUTE_PATH:
      if (value < 0 || value > 1) return fail(PDA_ERR_SHAPE, "compute path must be 0 or 1");
      g_compute_path.store(value);
      return PDA_OK;
    case PDA_OPT_FUSED_MERGE:
      if (value < 0 || value > 2) return fail(PDA_ERR_SHAPE, "fused merge must be 0, 1 or 2");
      g_fused_merge.store(value);
      return PDA_OK;
    case PDA_OPT_KV_GROUP:
      if (value < 0 || value > pda::kMaxWaves) return fail(PDA_ERR_SHAPE, "kv group must be in [0, %d]", pda::kMaxWaves);
      g_kv_group.store(value);
      return PDA_OK;
    case PDA_OPT_FIXED_SPLIT:
      if (value < 0 || value > 1) return fail(PDA_ERR_SHAPE, "fixed split must be 0 or 1");
      g_fixed_split.store(value);
      return PDA_OK;
    default:
      return fail(PDA_ERR_UNSUPPORTED, "unknown option %d", option);
  }
}

int32_t pda_get_option(int32_t option) {
  switch (option) {
    case PDA_OPT_BLOCKS_PER_CU: return blocks_per_cu();
    case PDA_OPT_MIN_STEPS: return min_steps_option();
    case PDA_OPT_COMPUTE_PATH: return compute_path();
    case PDA_OPT_FUSED_MERGE: return fused_merge();
    case PDA_OPT_KV_GROUP: return kv_group_cap();
    case PDA_OPT_FIXED_SPLIT: return fixed_split();
    default: return -1;
  }
}

int pda_stream_read(const void* buf, int64_t bytes, uint32_t* sink, int32_t unroll, int32_t blocks_per_cu,
                    void* stream) {
  g_err.clear();
  if (bytes <= 0 || bytes % 16) return fail(PDA_ERR_SHAPE, "bytes must be a positive multiple of 16");
  if (unroll == 0) unroll = 16;
  if (blocks_per_cu == 0) blocks_per_cu = 1;
  if (unroll != 4 && unroll != 8 && unroll != 16) return fail(PDA_ERR_UNSUPPORTED, "unroll must be 4, 8 or 16");
  if (blocks_per_cu < 1 || blocks_per_cu > 32) return fail(PDA_ERR_UNSUPPORTED, "blocks_per_cu must be in [1, 32]");
  if (!buf || !sink) return fail(PDA_ERR_NULL, "a pointer is NULL");
  if (reinterpret_cast<uintptr_t>(buf) & 15) return fail(PDA_ERR_ALIGN, "buf must be 16-byte aligned");
  if (reinterpret_cast<uintptr_t>(sink) & 3) return fail(PDA_ERR_ALIGN, "sink must be 4-byte aligned");
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  int cus = 0;
  int rc = device_cus(dev, &cus);
  if (rc) return rc;
  const int64_t blocks = static_cast<int64_t>(cus) * blocks_per_cu;
  if ((bytes + blocks - 1) / blocks > (int64_t{1} << 31) - 1024)
    return fail(PDA_ERR_SHAPE, "bytes too large for %lld workgroups", static_cast<long long>(blocks));
  e = pda::launch_stream_read(buf, bytes, sink, unroll, static_cast<int>(blocks), static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "stream read kernel launch");
  return PDA_OK;
}

int pda_profile_enable(int32_t on) {
  std::lock_guard<std::mutex> lock(g_prof_mu);
  g_prof_on = on != 0;
  return PDA_OK;
}

int pda_profile_read(double* split_ms, double* merge_ms, int64_t* calls) {
  g_err.clear();
  if (!split_ms || !merge_ms || !calls) return fail(PDA_ERR_NULL, "pda_profile_read: NULL output pointer");
  return prof_read(0, split_ms, merge_ms, calls);
}

int pda_profile_read_prelude(double* gemv_ms, double* epilogue_ms, int64_t* calls) {
  g_err.clear();
  if (!gemv_ms || !epilogue_ms || !calls) return fail(PDA_ERR_NULL, "pda_profile_read_prelude: NULL output pointer");
  return prof_read(1, gemv_ms, epilogue_ms, calls);
}

int pda_kv_append(const void* k_new, const void* v_new, void* k_cache, void* v_cache,
                  const int32_t* block_table, const int32_t* context_lens, int32_t batch, int32_t num_kv_heads,
                  int32_t head_dim, int32_t page_size, int32_t num_pages, int32_t max_pages_per_seq,
                  void* stream) {
  return pda_kv_append_n(k_new, v_new, k_cache, v_cache, block_table, context_lens, batch, 1, num_kv_heads,
                         head_dim, page_size, num_pages, max_pages_per_seq, stream);
}

int pda_kv_append_n(const void* k_new, const void* v_new, void* k_cache, void* v_cache,
                    const int32_t* block_table, const int32_t* context_lens, int32_t batch, int32_t num_tokens,
                    int32_t num_kv_heads, int32_t head_dim, int32_t page_size, int32_t num_pages,
                    int32_t max_pages_per_seq, void* stream) {
  g_err.clear();
  int rc = check_shape(batch, num_kv_heads, num_kv_heads, head_dim, page_size, max_pages_per_seq);
  if (rc) return rc;
  if (num_tokens < 1 || num_tokens > 1024)
    return fail(PDA_ERR_SHAPE, "num_tokens must be in [1, 1024] (got %d)", num_tokens);
  if (num_pages <= 0) return fail(PDA_ERR_SHAPE, "num_pages must be positive (got %d)", num_pages);
  if (batch == 0) return PDA_OK;
  if (!k_new || !v_new || !k_cache || !v_cache || !block_table || !context_lens)
    return fail(PDA_ERR_NULL, "a tensor pointer is NULL");
  auto misaligned = [](const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) != 0; };
  if (misaligned(k_new, 16) || misaligned(v_new, 16) || misaligned(k_cache, 16) || misaligned(v_cache, 16))
    return fail(PDA_ERR_ALIGN, "k_new, v_new, k_cache and v_cache must be 16-byte aligned");
  if (misaligned(block_table, 4) || misaligned(context_lens, 4))
    return fail(PDA_ERR_ALIGN, "block_table and context_lens must be 4-byte aligned");
  if ((rc = maybe_validate(block_table, context_lens, batch, max_pages_per_seq, page_size, num_pages,
                           static_cast<hipStream_t>(stream))))
    return rc;
  pda::AppendArgs a;
  a.k_new = static_cast<const uint16_t*>(k_new);
  a.v_new = static_cast<const uint16_t*>(v_new);
  a.k = static_cast<uint16_t*>(k_cache);
  a.v = static_cast<uint16_t*>(v_cache);
  a.bt = block_table;
  a.lens = context_lens;
  a.batch = batch;
  a.tokens = num_tokens;
  a.hkv = num_kv_heads;
  a.head_dim = head_dim;
  a.page_shift = log2i(page_size);
  a.num_pages = num_pages;
  a.maxp = max_pages_per_seq;
  hipError_t e = pda::launch_append_kernel(a, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "append kernel launch");
  return PDA_OK;
}

int paged_decode_attention_append(const void* q, const void* k_new, const void* v_new, void* k_cache,
                                  void* v_cache, const int32_t* block_table, const int32_t* context_lens,
                                  void* out, int32_t batch, int32_t num_q_heads, int32_t num_kv_heads,
                                  int32_t head_dim, int32_t page_size, int32_t num_pages,
                                  int32_t max_pages_per_seq, float scale, void* stream) {
  g_err.clear();
  // validate the attention arguments first so that nothing is written on error
  int rc = check_attention(batch, num_q_heads, num_kv_heads, head_dim, page_size, max_pages_per_seq);
  if (rc) return rc;
  if (!std::isfinite(scale)) return fail(PDA_ERR_SCALE, "scale is not finite");
  int valu_cols = 0;
  if ((rc = check_compute_path(head_dim, page_size, num_q_heads / num_kv_heads, batch, &valu_cols))) return rc;
  if (batch > 0 && (!q || !out)) return fail(PDA_ERR_NULL, "a tensor pointer is NULL");
  if ((reinterpret_cast<uintptr_t>(q) & 15) || (reinterpret_cast<uintptr_t>(out) & 15))
    return fail(PDA_ERR_ALIGN, "q, k_cache, v_cache and out must be 16-byte aligned");
  if ((rc = pda_kv_append(k_new, v_new, k_cache, v_cache, block_table, context_lens, batch, num_kv_heads,
                          head_dim, page_size, num_pages, max_pages_per_seq, stream)))
    return rc;
  return paged_decode_attention(q, k_cache, v_cache, block_table, context_lens, out, batch, num_q_heads,
                                num_kv_heads, head_dim, page_size, num_pages, max_pages_per_seq, scale, stream);
}

int paged_decode_attention(const void* q, const void* k_cache, const void* v_cache,
                           const int32_t* block_table, const int32_t* context_lens, void* out,
                           int32_t batch, int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
                           int32_t page_size, int32_t num_pages, int32_t max_pages_per_seq, float scale,
                           void* stream) {
  return paged_decode_attention_ext(q, k_cache, v_cache, block_table, context_lens, out, batch, num_q_heads,
                                    num_kv_heads, head_dim, page_size, num_pages, max_pages_per_seq, 1, 0,
                                    scale, stream);
}

int paged_decode_attention_ext(const void* q, const void* k_cache, const void* v_cache,
                               const int32_t* block_table, const int32_t* context_lens, void* out,
                               int32_t batch, int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
                               int32_t page_size, int32_t num_pages, int32_t max_pages_per_seq,
                               int32_t num_queries, int32_t window, float scale, void* stream) {
  return attention_call(q, k_cache, v_cache, block_table, context_lens, out, batch, num_q_heads, num_kv_heads,
                        head_dim, page_size, num_pages, max_pages_per_seq, num_queries, window, scale, stream,
                        false);
}

int paged_decode_attention_noalloc(const void* q, const void* k_cache, const void* v_cache,
                                   const int32_t* block_table, const int32_t* context_lens, void* out,
                                   int32_t batch, int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
                                   int32_t page_size, int32_t num_pages, int32_t max_pages_per_seq, float scale,
                                   void* stream) {
  return attention_call(q, k_cache, v_cache, block_table, context_lens, out, batch, num_q_heads, num_kv_heads,
                        head_dim, page_size, num_pages, max_pages_per_seq, 1, 0, scale, stream, true);
}

int paged_decode_attention_desc(const pda_tensor* q, const pda_tensor* k_cache, const pda_tensor* v_cache,
                                const pda_tensor* block_table, const pda_tensor* context_lens,
                                const pda_tensor* out, float scale, void* stream) {
  g_err.clear();
  const pda_tensor* ts[6] = {q, k_cache, v_cache, block_table, context_lens, out};
  static const char* const names[6] = {"q", "k_cache", "v_cache", "block_table", "context_lens", "out"};
  static const int32_t dtypes[6] = {PDA_DTYPE_BF16, PDA_DTYPE_BF16, PDA_DTYPE_BF16,
                                    PDA_DTYPE_I32,  PDA_DTYPE_I32,  PDA_DTYPE_BF16};
  static const int32_t ranks[6] = {3, 4, 4, 2, 1, 3};
  for (int i = 0; i < 6; ++i)
    if (!ts[i]) return fail(PDA_ERR_NULL, "%s: descriptor is NULL", names[i]);
  for (int i = 0; i < 6; ++i)
    if (ts[i]->dtype != dtypes[i])
      return fail(PDA_ERR_DTYPE, "%s: dtype %s (%d), expected %s", names[i], dtype_name(ts[i]->dtype),
                  ts[i]->dtype, dtype_name(dtypes[i]));
  int rc;
  for (int i = 0; i < 6; ++i)
    if ((rc = check_rank(*ts[i], names[i], ranks[i]))) return rc;
  const int64_t* qs = q->shape;
  const int64_t* ks = k_cache->shape;
  for (int i = 0; i < 3; ++i)
    if (out->shape[i] != qs[i]) return fail(PDA_ERR_SHAPE, "out must have the shape of q");
  for (int i = 0; i < 4; ++i)
    if (v_cache->shape[i] != ks[i]) return fail(PDA_ERR_SHAPE, "v_cache must have the shape of k_cache");
  if (ks[3] != qs[2])
    return fail(PDA_ERR_SHAPE, "head_dim of q (%lld) and of the caches (%lld) differ", static_cast<long long>(qs[2]),
                static_cast<long long>(ks[3]));
  if (block_table->shape[0] != qs[0] || context_lens->shape[0] != qs[0])
    return fail(PDA_ERR_SHAPE, "block_table and context_lens must have one row per sequence of q (%lld)",
                static_cast<long long>(qs[0]));
  for (int i = 0; i < 6; ++i)
    if ((rc = check_dense(*ts[i], names[i]))) return rc;
  for (int i = 0; i < 6; ++i)
    if (!desc_empty(*ts[i]) && !ts[i]->data) return fail(PDA_ERR_NULL, "%s: data is NULL", names[i]);
  return attention_call(q->data, k_cache->data, v_cache->data, static_cast<const int32_t*>(block_table->data),
                        static_cast<const int32_t*>(context_lens->data), out->data, static_cast<int32_t>(qs[0]),
                        static_cast<int32_t>(qs[1]), static_cast<int32_t>(ks[2]), static_cast<int32_t>(qs[2]),
                        static_cast<int32_t>(ks[1]), static_cast<int32_t>(ks[0]),
                        static_cast<int32_t>(block_table->shape[1]), 1, 0, scale, stream, false);
}

int pda_pack_weights(const void* w, void* w_packed, int32_t rows, int32_t cols, void* stream) {
  g_err.clear();
  if (rows <= 0 || cols <= 0) return fail(PDA_ERR_SHAPE, "rows and cols must be positive");
  if (rows % pda::kTileRows || cols % pda::kTileK)
    return fail(PDA_ERR_SHAPE, "rows must be a multiple of 16 and cols of 32 (got %d x %d)", rows, cols);
  if (static_cast<int64_t>(rows) * cols > (int64_t{1} << 34)) return fail(PDA_ERR_SHAPE, "matrix too large");
  if (!w || !w_packed) return fail(PDA_ERR_NULL, "a tensor pointer is NULL");
  if (misaligned(w, 16) || misaligned(w_packed, 16)) return fail(PDA_ERR_ALIGN, "w and w_packed must be 16-byte aligned");
  const uintptr_t a = reinterpret_cast<uintptr_t>(w), b = reinterpret_cast<uintptr_t>(w_packed);
  const uintptr_t bytes = static_cast<uintptr_t>(rows) * cols * 2;
  if (a < b + bytes && b < a + bytes) return fail(PDA_ERR_SHAPE, "w and w_packed overlap");
  hipError_t e = pda::launch_pack(static_cast<const uint16_t*>(w), static_cast<uint16_t*>(w_packed), rows, cols,
                                  static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_fail(e, "pack kernel launch");
  return PDA_OK;
}

int pda_attention_prelude(const void* x, const void* w_packed, const void* bias, const void* q_norm,
                          const void* k_norm, const int32_t* context_lens, void* q_out, void* k_out,
                          void* v_out, const pda_prelude_dims* dims, void* stream) {
  g_err.clear();
  int rc = check_prelude(dims);
  if (rc) return rc;
  if (dims->batch == 0) return PDA_OK;
  if (!k_out || !v_out) return fail(PDA_ERR_NULL, "a tensor pointer is NULL");
  if (misaligned(k_out, 16) || misaligned(v_out, 16))
    return fail(PDA_ERR_ALIGN, "x, w_packed and the outputs must be 16-byte aligned");
  pda::PreludeArgs ep{};
  ep.k_out = static_cast<uint16_t*>(k_out);
  ep.v_out = static_cast<uint16_t*>(v_out);
  return run_prelude(x, w_packed, bias, q_norm, k_norm, context_lens, q_out, ep, *dims, stream);
}

int pda_attention_prelude_append(const void* x, const void* w_packed, const void* bias, const void* q_norm,
                                 const void* k_norm, const int32_t* context_lens, void* q_out, void* k_cache,
                                 void* v_cache, const int32_t* block_table, int32_t page_size, int32_t num_pages,
                                 int32_t max_pages_per_seq, const pda_prelude_dims* dims, void* stream) {
  g_err.clear();
  int rc = check_prelude(dims);
  if (rc) return rc;
  if (page_size <= 0 || max_pages_per_seq <= 0)
    return fail(PDA_ERR_SHAPE, "page_size and max_pages_per_seq must be positive");
  if (!is_pow2(page_size) || page_size > PDA_MAX_PAGE_SIZE)
    return fail(PDA_ERR_UNSUPPORTED, "page_size %d (supported: powers of two up to %d)", page_size,
                PDA_MAX_PAGE_SIZE);
  if (static_cast<int64_t>(max_pages_per_seq) * page_size > (int64_t{1} << 30))
    return fail(PDA_ERR_SHAPE, "max_pages_per_seq * page_size too large");
  if (num_pages <= 0) return fail(PDA_ERR_SHAPE, "num_pages must be positive (got %d)", num_pages);
  if (dims->batch == 0) return PDA_OK;
  if (!k_cache || !v_cache || !block_table) return fail(PDA_ERR_NULL, "a tensor pointer is NULL");
  if (misaligned(k_cache, 16) || misaligned(v_cache, 16) || misaligned(block_table, 4))
    return fail(PDA_ERR_ALIGN, "caches must be 16-byte and block_table 4-byte aligned");
  pda::PreludeArgs ep{};
  ep.k_cache = static_cast<uint16_t*>(k_cache);
  ep.v_cache = static_cast<uint16_t*>(v_cache);
  ep.bt = block_table;
  ep.page_shift = log2i(page_size);
  ep.num_pages = num_pages;
  ep.maxp = max_pages_per_seq;
  return run_prelude(x, w_packed, bias, q_norm, k_norm, context_lens, q_out, ep, *dims, stream);
}

int pda_o_proj_residual_norm(const void* attn, const void* w_packed, const void* residual, const void* norm_w,
                             void* residual_out, void* normed_out, int32_t batch, int32_t in_features,
                             int32_t hidden, float eps, void* stream) {
  g_err.clear();
  if (batch < 0) return fail(PDA_ERR_SHAPE, "batch must be >= 0 (got %d)", batch);
  if (batch > pda::kMaxGemvBatch) return fail(PDA_ERR_UNSUPPORTED, "batch %d exceeds %d", batch, pda::kMaxGemvBatch);
  if (in_features <= 0 || hidden <= 0) return fail(PDA_ERR_SHAPE, "in_features and hidden must be positive");
  if (in_features % pda::kTileK || in_features > 65536)
    return fail(PDA_ERR_UNSUPPORTED, "in_features %d (supported: multiples of 32 up to 65536)", in_features);
  if (hidden % pda::kTileRows || hidden > pda::kMaxOProjHidden)
    return fail(PDA_ERR_UNSUPPORTED, "hidden %d (supported: multiples of 16 up to %d)", hidden,
                pda::kMaxOProjHidden);
  if (batch > pda::kMaxGemvBatchAnyRows && hidden % 128)
    return fail(PDA_ERR_UNSUPPORTED, "o_proj batch %d above %d needs hidden a multiple of 128", batch,
                pda::kMaxGemvBatchAnyRows);
  if (!std::isfinite(eps) || eps < 0.f) return fail(PDA_ERR_SCALE, "eps must be finite and >= 0");
  if (batch == 0) return PDA_OK;
  if (!attn || !w_packed || !residual || !norm_w || !residual_out || !normed_out)
    return fail(PDA_ERR_NULL, "a tensor pointer is NULL");
  if (misaligned(attn, 16) || misaligned(w_packed, 16))
    return fail(PDA_ERR_ALIGN, "attn and w_packed must be 16-byte aligned");
  if (misaligned(residual, 2) || misaligned(norm_w, 2) || misaligned(residual_out, 2) || misaligned(normed_out, 2))
    return fail(PDA_ERR_ALIGN, "bf16 arrays must be 2-byte aligned");
  if (normed_out == residual_out) return fail(PDA_ERR_SHAPE, "normed_out must not be residual_out");
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  int cus = 0;
  int rc = device_cus(dev, &cus);
  if (rc) return rc;
  hipStream_t st = static_cast<hipStream_t>(stream);
  const pda::GemvPlan plan = pda::plan_gemv(batch, hidden, in_features, cus, /*seq_major=*/true);
  void* ws = nullptr;
  if ((rc = workspace_for(dev, st, oproj_ws_bytes(plan, batch, hidden), &ws))) return rc;
  pda::GemvArgs g;
  g.x = static_cast<const uint16_t*>(attn);
  g.wp = static_cast<const uint16_t*>(w_packed);
  g.part = static_cast<float*>(ws);
  g.batch = batch;
  g.n = hidden;
  g.k = in_features;
  g.plan = plan;
  const Rec rec = prof_begin(2);
  const bool prof = rec.a != nullptr;
  if (prof && (e = hipEventRecord(rec.a, st)) != hipSuccess) return hip_fail(e, "hipEventRecord");
  if ((e = pda::launch_gemv(g, st)) != hipSuccess) return hip_fail(e, "GEMV kernel launch");
  if (prof && (e = hipEventRecord(rec.b, st)) != hipSuccess) return hip_fail(e, "hipEventRecord");
  pda::OProjArgs o;
  o.part = g.part;
  o.plan = plan;
  o.residual = static_cast<const uint16_t*>(residual);
  o.norm_w = static_cast<const uint16_t*>(norm_w);
  o.residual_out = static_cast<uint16_t*>(residual_out);
  o.normed_out = static_cast<uint16_t*>(normed_out);
  o.z = reinterpret_cast<float*>(static_cast<char*>(ws) + oproj_z_offset(plan, batch, hidden));
  o.chunk_ss = o.z + static_cast<int64_t>(batch) * hidden;
  o.batch = batch;
  o.hidden = hidden;
  o.eps = eps;
  if ((e = pda::launch_oproj_epilogue(o, st)) != hipSuccess) return hip_fail(e, "o_proj epilogue launch");
  if (prof) {
    if ((e = hipEventRecord(rec.c, st)) != hipSuccess) return hip_fail(e, "hipEventRecord");
    prof_push(rec);
  }
  return PDA_OK;
}

int pda_o_proj_workspace_reserve(int32_t batch, int32_t in_features, int32_t hidden, void* stream) {
  g_err.clear();
  if (batch < 0 || batch > pda::kMaxGemvBatch || in_features <= 0 || in_features % pda::kTileK ||
      hidden <= 0 || hidden % pda::kTileRows || hidden > pda::kMaxOProjHidden ||
      (batch > pda::kMaxGemvBatchAnyRows && hidden % 128))
    return fail(PDA_ERR_SHAPE, "o_proj shape out of range");
  if (batch == 0) return PDA_OK;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  int cus = 0;
  int rc = device_cus(dev, &cus);
  if (rc) return rc;
  const pda::GemvPlan plan = pda::plan_gemv(batch, hidden, in_features, cus, /*seq_major=*/true);
  void* ptr = nullptr;
  return workspace_for(dev, static_cast<hipStream_t>(stream), oproj_ws_bytes(plan, batch, hidden), &ptr);
}

int pda_profile_read_o_proj(double* gemv_ms, double* epilogue_ms, int64_t* calls) {
  g_err.clear();
  if (!gemv_ms || !epilogue_ms || !calls) return fail(PDA_ERR_NULL, "pda_profile_read_o_proj: NULL output pointer");
  return prof_read(2, gemv_ms, epilogue_ms, calls);
}

int pda_validate_paging(const int32_t* block_table, const int32_t* context_lens, int32_t batch,
                        int32_t max_pages_per_seq, int32_t page_size, int32_t num_pages, void* stream) {
  g_err.clear();
  if (batch < 0 || max_pages_per_seq <= 0 || page_size <= 0 || num_pages <= 0)
    return fail(PDA_ERR_SHAPE, "batch, max_pages_per_seq, page_size and num_pages out of range");
  if (batch == 0) return PDA_OK;
  if (!block_table || !context_lens) return fail(PDA_ERR_NULL, "a tensor pointer is NULL");
  if (static_cast<int64_t>(batch) * max_pages_per_seq > (int64_t{1} << 31))
    return fail(PDA_ERR_SHAPE, "block_table too large to validate");
  return validate_paging(block_table, context_lens, batch, max_pages_per_seq, page_size, num_pages,
                         static_cast<hipStream_t>(stream));
}

int pda_prelude_workspace_reserve(const pda_prelude_dims* dims, void* stream) {
  g_err.clear();
  int rc = check_prelude(dims);
  if (rc) return rc;
  if (dims->batch == 0) return PDA_OK;
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  int cus = 0;
  if ((rc = device_cus(dev, &cus))) return rc;
  void* ptr = nullptr;
  return workspace_for(dev, static_cast<hipStream_t>(stream), prelude_ws_bytes(*dims, cus), &ptr);
}

}  // extern "C"
