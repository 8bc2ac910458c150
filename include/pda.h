/*
 * pda.h -- paged decode attention for AMD MI355X (gfx950), C ABI.
 *
 * The operation is the decode-attention body of the paper's kernel family
 * (iv) (Method, "Principle-Driven LLM Kernel Generator"): one query token per
 * sequence attends over that sequence's cached keys and values, which live in
 * fixed-size pages of a shared pool addressed through a per-sequence page
 * table (the paged KV cache of Method, "Kernel Customization and
 * Multi-Request Adaptation").  The work is split along the context across
 * many waves, each running an online softmax over its share, and the
 * per-split results are merged with a log-sum-exp combination (the paper's
 * "cross-CTA merging"; the appendix describes its hand-written reference as
 * merging without a separate reduction kernel).
 *
 * For sequence b with L_b cached tokens and query head h (kv head
 * g = h / G, G = num_q_heads / num_kv_heads):
 *     s_t        = scale * <q[b,h,:], K[page(b,t), t % P, g, :]>
 *     out[b,h,:] = sum_t softmax(s)_t * V[page(b,t), t % P, g, :]
 *     page(b,t)  = block_table[b, t / P],   t = 0 .. L_b - 1
 * L_b counts every cached token including the one appended for the current
 * step (the paper advances the length by one after its KV append).  A
 * sequence with L_b = 0 gets a zero output row.
 *
 * Arithmetic: bf16 inputs, fp32 accumulation (scores, running max and sum,
 * the probability-times-value products on bf16 matrix cores with each
 * probability carried as a sum of two bf16 values, ~2^-17 relative), bf16
 * round-to-nearest-even output.  Scores are formed in fp32: scale * q.k must
 * stay within the fp32 range.
 *
 * Memory: every pointer argument of paged_decode_attention is a DEVICE
 * pointer on the current HIP device.  The caller allocates and owns all of
 * them; the library never frees or retains them.  The library owns one
 * internal workspace per (device, stream), grown on demand (see
 * pda_workspace_reserve) and released by pda_release_workspaces.
 *
 * Interface readings: the paper defines the operations (attention, its KV
 * append, prelude and output projection), not a library interface.  Calls
 * marked [library interface] below -- workspace management, planning,
 * options, validation, timing, error reporting -- are this library's own,
 * with no counterpart in the paper; so are the status codes and their
 * numbering.
 *
 * Errors: every entry point returns PDA_OK (0) or a PDA_ERR_* code and sets a
 * thread-local message readable with pda_last_error().  Argument checks run
 * before any HIP call; on an argument error nothing is launched and `out` is
 * untouched.  Device-resident contents are not validated: page ids outside
 * [0, num_pages) are clamped into range and lengths are clamped to
 * [0, max_pages_per_seq * page_size], so bad contents give unspecified
 * values but never an out-of-bounds access.
 */
#ifndef PDA_H
#define PDA_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define PDA_VERSION 1

enum pda_status {
  PDA_OK = 0,
  PDA_ERR_NULL = 1,        /* a required pointer is NULL                          */
  PDA_ERR_SHAPE = 2,       /* a size is out of range or inconsistent              */
  PDA_ERR_UNSUPPORTED = 3, /* valid but not implemented (head_dim, group, page)   */
  PDA_ERR_SCALE = 4,       /* scale is not a finite number                        */
  PDA_ERR_ALIGN = 5,       /* q, k_cache, v_cache or out not 16-byte aligned      */
  PDA_ERR_HIP = 6,         /* a HIP runtime call failed (message has the detail)  */
  PDA_ERR_DTYPE = 7,       /* a tensor descriptor has the wrong element type      */
  PDA_ERR_LAYOUT = 8       /* a tensor descriptor's strides are not the layout
                              the operation reads (see pda_tensor)                */
};

/* Supported set of this version. */
#define PDA_MAX_BATCH 8192
#define PDA_MAX_BATCH_D256 4096  /* attention at head_dim 256: the kernel's
                                    per-sequence table shares LDS with its
                                    34 KB-per-wave K/V tiles                */
#define PDA_MAX_GROUP 16      /* num_q_heads / num_kv_heads                */
#define PDA_MAX_PAGE_SIZE 1024
#define PDA_MAX_KV_HEADS 1024

/*
 * paged_decode_attention -- the decode-attention step described above.
 *
 *   q            bf16 [batch, num_q_heads, head_dim], contiguous, 16-B aligned.
 *   k_cache      bf16 [num_pages, page_size, num_kv_heads, head_dim],
 *                contiguous, 16-B aligned (token-major pages; the kv heads of
 *                one token are adjacent).
 *   v_cache      same shape and layout as k_cache.
 *   block_table  int32 [batch, max_pages_per_seq], row-major.  Only the first
 *                ceil(L_b / page_size) entries of row b are read.
 *   context_lens int32 [batch], on the device (no host read, so the call can
 *                be captured in a HIP graph).
 *   out          bf16 [batch, num_q_heads, head_dim], contiguous, 16-B
 *                aligned; fully written on success.  Must not alias inputs.
 *   head_dim     64, 128 or 256.   page_size: a power of two in [1, 1024].
 *   num_q_heads  a multiple of num_kv_heads, with group <= 16.
 *   batch        0 .. 8192 (0 is a no-op); at head_dim 256, 0 .. 4096.
 *   scale        finite fp32 multiplier of the scores (usually 1/sqrt(D)).
 *   stream       hipStream_t to launch on; NULL means the null stream.
 *
 * Asynchronous: returns after enqueueing; no host synchronisation.  Calls on
 * one stream are ordered; calls on different streams use separate
 * workspaces.  If the stream is being captured, the workspace must already
 * be large enough (pda_workspace_reserve), otherwise PDA_ERR_HIP.
 */
int paged_decode_attention(const void* q, const void* k_cache, const void* v_cache,
                           const int32_t* block_table, const int32_t* context_lens,
                           void* out,
                           int32_t batch, int32_t num_q_heads, int32_t num_kv_heads,
                           int32_t head_dim, int32_t page_size, int32_t num_pages,
                           int32_t max_pages_per_seq,
                           float scale, void* stream);

/*
 * Tensor descriptors: the dtype and layout half of the contract, for callers
 * that hold tensors rather than bare pointers.  The paper's contract for a
 * generated kernel names the tensor interface and its dtype rules (Problem
 * Formulation, the contract-gated tier); its attention operates on bf16
 * models (Experiments, Setup).  The descriptor form checks both before any
 * HIP call:
 *   data    device pointer of element [0, 0, ...].
 *   dtype   a pda_dtype.
 *   ndim    dimensions in use (1 .. PDA_MAX_DIMS); shape[i], stride[i] for
 *           i < ndim, strides in elements.
 * The attention reads dense row-major tensors: stride[ndim - 1] = 1 and
 * stride[i] = stride[i + 1] * shape[i + 1]; the stride of a dimension of
 * extent 1 is not looked at, and an empty tensor has no layout.  Other
 * strides (transposed, sliced or padded views) give PDA_ERR_LAYOUT.
 */
typedef enum {
  PDA_DTYPE_BF16 = 0,
  PDA_DTYPE_F16 = 1,
  PDA_DTYPE_F32 = 2,
  PDA_DTYPE_I32 = 3,
  PDA_DTYPE_I64 = 4
} pda_dtype;

#define PDA_MAX_DIMS 4
typedef struct {
  void* data;
  int32_t dtype;
  int32_t ndim;
  int64_t shape[PDA_MAX_DIMS];
  int64_t stride[PDA_MAX_DIMS];
} pda_tensor;

/*
 * paged_decode_attention_desc -- paged_decode_attention with tensor
 * descriptors:
 *   q, out        PDA_DTYPE_BF16, ndim 3: [batch, num_q_heads, head_dim]
 *   k_cache       PDA_DTYPE_BF16, ndim 4: [num_pages, page_size, num_kv_heads, head_dim]
 *   v_cache       same dtype and shape as k_cache
 *   block_table   PDA_DTYPE_I32, ndim 2: [batch, max_pages_per_seq]
 *   context_lens  PDA_DTYPE_I32, ndim 1: [batch]
 * all dense row-major.  The sizes come from the shapes; everything else
 * (semantics, supported set, alignment, workspace, asynchrony, capture) is
 * as for paged_decode_attention.  Errors, all before any HIP call:
 *   PDA_ERR_NULL    a descriptor is NULL, or a non-empty tensor's data is NULL;
 *   PDA_ERR_DTYPE   a dtype other than the one listed (fp16, fp32 or int64
 *                   tensors are not converted);
 *   PDA_ERR_SHAPE   an ndim other than the one listed, a negative extent, or
 *                   shapes that disagree (out vs q, v_cache vs k_cache,
 *                   head_dim of q vs the caches, batch of block_table and
 *                   context_lens vs q, num_q_heads not a multiple of
 *                   num_kv_heads) or exceed int32;
 *   PDA_ERR_LAYOUT  strides other than the dense row-major ones;
 *   then the checks of paged_decode_attention (PDA_ERR_UNSUPPORTED for
 *   head_dim, page_size or group, PDA_ERR_SCALE, PDA_ERR_ALIGN, ...).
 */
int paged_decode_attention_desc(const pda_tensor* q, const pda_tensor* k_cache, const pda_tensor* v_cache,
                                const pda_tensor* block_table, const pda_tensor* context_lens,
                                const pda_tensor* out, float scale, void* stream);

/*
 * paged_decode_attention_ext -- the same step with a key range per query:
 * several query tokens per sequence and an optional sliding window.  The
 * paper's engine mixes chunked prefill with decode steps (Method, "Kernel
 * Customization and Multi-Request Adaptation") and adapts attention to a
 * sliding window for Mistral (its table of model-specific adaptations); it
 * defines neither, so this is the reading implemented:
 *
 *   q, out        bf16 [batch, num_queries, num_q_heads, head_dim], contiguous.
 *                 The num_queries query tokens are the sequence's last ones:
 *                 query j sits at position L_b - num_queries + j and sees keys
 *                 t <= that position (causal).  The new tokens must already be
 *                 in the cache and counted in context_lens.
 *   window        0: no window.  W > 0: the query at position p sees only
 *                 keys p - W < t <= p (W keys, its own included).  Pages that
 *                 lie wholly before the first key any query of the sequence
 *                 sees are never read: their block_table entries may be stale
 *                 or -1.
 *   num_queries   1 .. 16, with num_queries * (num_q_heads / num_kv_heads) <= 16
 *                 (one matrix-core column per query token and head);
 *                 otherwise PDA_ERR_UNSUPPORTED.
 * A query that sees no key (L_b < num_queries, or L_b = 0) gets a zero row.
 * Everything else -- layout, ownership, errors, workspace, capture -- is as
 * for paged_decode_attention, which is this call with num_queries = 1 and
 * window = 0.
 */
int paged_decode_attention_ext(const void* q, const void* k_cache, const void* v_cache,
                               const int32_t* block_table, const int32_t* context_lens, void* out,
                               int32_t batch, int32_t num_q_heads, int32_t num_kv_heads,
                               int32_t head_dim, int32_t page_size, int32_t num_pages,
                               int32_t max_pages_per_seq, int32_t num_queries, int32_t window,
                               float scale, void* stream);

/*
 * pda_kv_append -- write each sequence's newest key and value into its page:
 * the step before attention in the paper's decode loop (Method, "Kernel
 * Customization and Multi-Request Adaptation": a small scatter kernel writes
 * the new K/V vectors and attention then runs with the sequence length
 * advanced by one).
 *
 *   k_new, v_new  bf16 [batch, num_kv_heads, head_dim], contiguous, 16-B aligned.
 *   k_cache, v_cache, block_table, num_pages, page_size, max_pages_per_seq
 *                 as for paged_decode_attention; the caches are written in place.
 *   context_lens  int32 [batch] on the device, already counting the new token:
 *                 sequence b's vectors go to position L_b - 1, i.e. page
 *                 block_table[b, (L_b-1) / page_size], slot (L_b-1) % page_size,
 *                 every kv head.  L_b = 0 writes nothing.
 * Only those slots change.  Two sequences whose page tables send their new
 * token to the same slot race (the page table must not do that).
 * Asynchronous on `stream`; no workspace, no allocation (graph-capturable).
 * Errors as for paged_decode_attention.
 */
int pda_kv_append(const void* k_new, const void* v_new, void* k_cache, void* v_cache,
                  const int32_t* block_table, const int32_t* context_lens,
                  int32_t batch, int32_t num_kv_heads, int32_t head_dim, int32_t page_size,
                  int32_t num_pages, int32_t max_pages_per_seq, void* stream);

/*
 * pda_kv_append_n -- the same for num_tokens (1 .. 1024) new tokens per
 * sequence, as a step of several query tokens needs (paged_decode_attention_ext):
 * k_new, v_new bf16 [batch, num_tokens, num_kv_heads, head_dim]; the lengths
 * count all of them and token j of sequence b lands at position
 * L_b - num_tokens + j; positions below 0 (L_b < num_tokens) write nothing.
 * pda_kv_append is this call with num_tokens = 1.
 */
int pda_kv_append_n(const void* k_new, const void* v_new, void* k_cache, void* v_cache,
                    const int32_t* block_table, const int32_t* context_lens, int32_t batch, int32_t num_tokens,
                    int32_t num_kv_heads, int32_t head_dim, int32_t page_size, int32_t num_pages,
                    int32_t max_pages_per_seq, void* stream);

/*
 * paged_decode_attention_append -- pda_kv_append followed by
 * paged_decode_attention on the same stream: append the step's key/value,
 * then attend with the length that counts them.  Arguments as for the two
 * calls; q and out as for paged_decode_attention.
 */
int paged_decode_attention_append(const void* q, const void* k_new, const void* v_new,
                                  void* k_cache, void* v_cache, const int32_t* block_table,
                                  const int32_t* context_lens, void* out,
                                  int32_t batch, int32_t num_q_heads, int32_t num_kv_heads,
                                  int32_t head_dim, int32_t page_size, int32_t num_pages,
                                  int32_t max_pages_per_seq, float scale, void* stream);

/*
 * paged_decode_attention_noalloc -- paged_decode_attention for callers that
 * cannot allocate device memory: code under HIP graph capture, tight serving
 * loops and harnesses that forbid hipMalloc.  Same operation, arguments,
 * layouts and errors, and the same kernels; the split partials, the steps
 * prefix and the split list go to a fixed buffer the library holds on each
 * device it runs on (a static device array of PDA_NOALLOC_SCRATCH_BYTES,
 * kept until the process ends) instead of the per-(device, stream)
 * workspace.  The call makes no hipMalloc or hipFree and needs no
 * pda_workspace_reserve; the caller still passes every input and output.
 *   - A shape whose plan needs more than PDA_NOALLOC_SCRATCH_BYTES fails
 *     with PDA_ERR_UNSUPPORTED before any launch.  pda_plan's
 *     workspace_bytes bounds the need (it covers 16 query columns per kv
 *     head; one query token needs G).
 *   - Every call on one device shares that device's buffer: two calls whose
 *     executions overlap on one device (different streams, or graphs
 *     replayed concurrently) race and give wrong results.  Order them.
 *   - The buffer keeps the last call's contents; nothing in it needs to
 *     start at any value.
 *   - PDA_DEBUG_VALIDATE and the kernel timing (pda_profile_enable) do not
 *     apply to this entry point.
 */
#define PDA_NOALLOC_SCRATCH_BYTES (64 * 1024 * 1024)
int paged_decode_attention_noalloc(const void* q, const void* k_cache, const void* v_cache,
                                   const int32_t* block_table, const int32_t* context_lens, void* out,
                                   int32_t batch, int32_t num_q_heads, int32_t num_kv_heads,
                                   int32_t head_dim, int32_t page_size, int32_t num_pages,
                                   int32_t max_pages_per_seq, float scale, void* stream);

/*
 * pda_plan [library interface] -- host-only dry run of the split planner: how the context of the
 * batch is spread over waves (the paper's split across CTAs, sized here to
 * fill the given number of compute units).  No HIP call.
 *   num_cus      compute units of the target device (256 on MI355X).
 *   grid_blocks  out: workgroups of the split kernel (one query token per
 *                sequence, the plan paged_decode_attention makes).
 *   waves        out: waves (workers) in that grid.
 *   workspace_bytes out: device workspace a call with this shape may need,
 *                for any num_queries of paged_decode_attention_ext.
 * Returns PDA_OK or an argument error as paged_decode_attention would.
 */
int pda_plan(int32_t batch, int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
             int32_t page_size, int32_t max_pages_per_seq, int32_t num_cus,
             int32_t* grid_blocks, int32_t* waves, int64_t* workspace_bytes);

/*
 * pda_workspace_reserve [library interface] -- grow the workspace of (current device, stream) so
 * that a later call with this shape (any num_queries and window) allocates
 * nothing (e.g. before graph capture).  Synchronous; may call hipMalloc.
 * A graph captured on a stream keeps using the workspace it was captured
 * with: reserve the largest shape before capturing, and neither grow that
 * stream's workspace (a larger eager call on the same stream) nor release it
 * (pda_release_workspaces) while the graph may still be replayed.
 */
int pda_workspace_reserve(int32_t batch, int32_t num_q_heads, int32_t num_kv_heads,
                          int32_t head_dim, int32_t page_size, int32_t max_pages_per_seq,
                          void* stream);

/* [library interface] Free every workspace the library holds (synchronises
   their streams). */
int pda_release_workspaces(void);

/*
 * Threads: calls may come from several host threads; error messages are
 * per thread.  The workspace belongs to a (device, stream) pair, so calls on
 * one stream must not be issued from two host threads at the same time.
 */

/*
 * pda_validate_paging [library interface] -- debugging aid: synchronise `stream`, copy
 * context_lens [batch] and block_table [batch, max_pages_per_seq] (device
 * pointers) to the host and check 0 <= L_b <= max_pages_per_seq * page_size
 * and 0 <= block_table[b][j] < num_pages for every page a sequence uses.
 * Returns PDA_OK, or PDA_ERR_SHAPE naming the first bad entry.  The kernels
 * never trust these device contents (out-of-range values are clamped, so a
 * bad table gives wrong numbers but no fault); with PDA_DEBUG_VALIDATE=1 in
 * the environment, every attention and append call runs this check first
 * (synchronising; skipped while the stream is being captured).
 */
int pda_validate_paging(const int32_t* block_table, const int32_t* context_lens, int32_t batch,
                        int32_t max_pages_per_seq, int32_t page_size, int32_t num_pages, void* stream);

/* [library interface] Thread-local message of the last failing call on this
   thread ("" if none). */
const char* pda_last_error(void);

/* [library interface] PDA_VERSION of the built library. */
int32_t pda_version(void);

/*
 * Planner options [library interface] (tuning and testing).  The split planner spreads the
 * batch's context over min(num_cus * blocks_per_cu, ceil(total 32-token
 * steps / (min_steps * step phases))) workgroups of up to 8 waves.
 *   PDA_OPT_BLOCKS_PER_CU  workgroups per compute unit, 1..8
 *                          (default 1, env PDA_BLOCKS_PER_CU).
 *   PDA_OPT_MIN_STEPS      fewest 32-token steps a wave is given, >= 1,
 *                          or 0 = the planner's choice (default, env
 *                          PDA_MIN_STEPS): 2, or 1 for a call whose K and V
 *                          (bounded by the page table) fit in 128 MB and
 *                          whose 2-step plan has several workgroups but
 *                          fewer than the device's CUs.  A large value
 *                          forces fewer splits, 1 the most.
 *   PDA_OPT_COMPUTE_PATH   where the attention kernel forms QK^T and P.V:
 *                          0 = matrix cores (default, env PDA_COMPUTE_PATH),
 *                          1 = vector ALU (bf16 dot2 products, DPP
 *                          reductions across lanes, fp32 FMAs for P.V).
 *                          Path 1 exists to measure the matrix-core choice
 *                          against: it takes head_dim 128, page_size >= 16
 *                          and at most 8 (query token, head) columns per kv
 *                          head; other shapes fail with PDA_ERR_UNSUPPORTED
 *                          while it is selected.  Outputs of the two paths
 *                          agree within the attention tolerance, not bitwise.
 *   PDA_OPT_FUSED_MERGE    0 (default, env PDA_FUSED_MERGE): split
 *                          sequences are merged by a second kernel.
 *                          1: plans with little partial data per sequence
 *                          (small batches, single requests) merge inside
 *                          the attention kernel, by the last workgroup to
 *                          finish each sequence: a call that takes the
 *                          fixed split keeps it (the pieces of a sequence
 *                          follow from its length), a stream-K plan takes
 *                          one kv head per workgroup if that is what it
 *                          takes (both measured slower than the merge
 *                          kernel on MI355X: the in-kernel hand-off costs
 *                          more than a launch);
 *                          2: every plan with several workgroups merges in
 *                          the attention kernel, with the default kv-head
 *                          grouping (for tests: slow for long contexts).
 *                          All are deterministic for a fixed plan; they
 *                          round differently.
 *   PDA_OPT_KV_GROUP       most kv heads a workgroup reads together, 0..8
 *                          (default 0 = the planner's choice, env
 *                          PDA_KV_GROUP): the largest divisor of
 *                          num_kv_heads not above it.  Fewer heads per
 *                          workgroup mean smaller partials per split piece
 *                          and shorter token rows read at a time.  The
 *                          planner takes 8 (4 above 8 columns per kv head),
 *                          and for a call whose K and V fit in 128 MB the
 *                          largest group that cuts no (sequence, kv-head
 *                          group) into more than 32 pieces.
 *   PDA_OPT_FIXED_SPLIT    1 (default, env PDA_FIXED_SPLIT): a call whose
 *                          K and V fit in 128 MB and that has at most half
 *                          the device's workgroups' worth of (sequence,
 *                          kv-head group) pairs cuts every pair into the
 *                          same number of chunks of whole 32-token steps
 *                          sized by the page table's largest context, so
 *                          that a workgroup knows its piece from its index
 *                          (no steps prefix on the way to the first loads;
 *                          the merge finds the pieces from the lengths).
 *                          Where the stream-K plan would take a single
 *                          workgroup, every pair is one chunk: whole
 *                          sequences on separate workgroups, no merge.
 *                          0: every call is split stream-K over the actual
 *                          lengths.  Both are deterministic for a fixed
 *                          plan; they round differently.
 * Options are process-wide and apply to later calls.  pda_set_option
 * returns PDA_OK or PDA_ERR_SHAPE / PDA_ERR_UNSUPPORTED; pda_get_option
 * returns the current value or -1 for an unknown option.
 */
#define PDA_OPT_BLOCKS_PER_CU 1
#define PDA_OPT_MIN_STEPS 2
#define PDA_OPT_COMPUTE_PATH 3
#define PDA_OPT_FUSED_MERGE 4
#define PDA_OPT_KV_GROUP 5
#define PDA_OPT_FIXED_SPLIT 6
int pda_set_option(int32_t option, int32_t value);
int32_t pda_get_option(int32_t option);

/*
 * Kernel timing [library interface] for measurement harnesses.  While enabled, every attention
 * call (paged_decode_attention and its _ext / _append forms) and every
 * prelude call records HIP events on its stream around each kernel it
 * launches.  pda_profile_read synchronises those events, returns
 * the summed milliseconds of the split kernel and of the merge kernel and
 * the number of calls recorded since the last read, and clears the record.
 */
int pda_profile_enable(int32_t on);
int pda_profile_read(double* split_ms, double* merge_ms, int64_t* calls);
/* The same for the prelude and o_proj calls: summed GEMV and epilogue ms. */
int pda_profile_read_prelude(double* gemv_ms, double* epilogue_ms, int64_t* calls);
int pda_profile_read_o_proj(double* gemv_ms, double* epilogue_ms, int64_t* calls);

/*
 * Streaming-read reference [library interface] for measurement harnesses: one kernel that only
 * reads `bytes` of device memory at `buf` (16-byte aligned, bytes a positive
 * multiple of 16), each byte once, with the attention kernel's loads
 * (16-byte non-temporal buffer loads).  Its bandwidth is what an HBM-bound
 * kernel can reach on this GPU, beside the 8 TB/s specification.
 *   sink           device uint32 the kernel writes only if the data XOR-folds
 *                  to one fixed value (it keeps the reads from being
 *                  optimised away); caller-owned
 *   unroll         16-byte loads in flight per lane: 4, 8 or 16 (0 = 16)
 *   blocks_per_cu  workgroups of 4 waves per compute unit, 1 .. 32 (0 = 1)
 * Asynchronous on `stream` (NULL = default); time it with events.  Returns
 * PDA_OK, PDA_ERR_NULL, PDA_ERR_SHAPE (bytes), PDA_ERR_ALIGN,
 * PDA_ERR_UNSUPPORTED (unroll, blocks_per_cu) or PDA_ERR_HIP.
 */
int pda_stream_read(const void* buf, int64_t bytes, uint32_t* sink, int32_t unroll, int32_t blocks_per_cu,
                    void* stream);

/*
 * ---------------------------------------------------------------------------
 * Attention prelude: the paper's kernel family (i) (Method, "Principle-Driven
 * LLM Kernel Generator"): the QKV projection of the new token's hidden
 * state plus rotary position embedding, optionally with a per-head RMSNorm
 * of q and k, producing this decode step's q, k and v.
 *
 *   y = W x (+ bias), W [N, H] with N = (Hq + 2 Hkv) * D, rows ordered q
 *   heads, k heads, v heads; each q and k head t (D values) becomes
 *   t / sqrt(mean(t^2) + eps) * w when norm weights are given, and then
 *   pair i < rotary_dim / 2 turns by the angle p * theta^(-2 i / rotary_dim),
 *   p = max(context_lens[b] - 1, 0) (the position of the new token; the
 *   length counts it): (a, b) -> (a cos - b sin, b cos + a sin), with pairs
 *   (i, i + rotary_dim / 2), or (2i, 2i + 1) when interleaved; dimensions at
 *   or beyond rotary_dim pass through.  v is only projected.  Intermediates
 *   stay fp32 (angles fp64); outputs are rounded once to bf16.
 * ---------------------------------------------------------------------------
 */
typedef struct {
  int32_t batch;         /* sequences, 0 .. 256; above 64, (num_q_heads +
                            2 num_kv_heads) * head_dim a multiple of 128       */
  int32_t hidden;        /* H: a positive multiple of 32, at most 65536         */
  int32_t num_q_heads;   /* Hq, a multiple of num_kv_heads                      */
  int32_t num_kv_heads;  /* Hkv                                                 */
  int32_t head_dim;      /* D: 64, 128 or 256                                   */
  int32_t rotary_dim;    /* 0 (no rotation) or even, 2 .. head_dim              */
  int32_t interleaved;   /* 0: pairs (i, i + rotary_dim/2); 1: pairs (2i, 2i+1) */
  float rope_theta;      /* base of the rotary frequencies, finite and > 0      */
  float eps;             /* RMSNorm epsilon, finite and >= 0                    */
} pda_prelude_dims;

/*
 * pda_pack_weights [library interface] -- copy a bf16 [rows, cols] row-major weight matrix into
 * the packed order the prelude reads (16-row x 32-column tiles of 1 KB in
 * matrix-core operand order).  rows a multiple of 16, cols a multiple of 32;
 * w and w_packed (rows * cols bf16, caller-owned, not overlapping) 16-byte
 * aligned.  Asynchronous on `stream`; done once per weight at load time.
 */
int pda_pack_weights(const void* w, void* w_packed, int32_t rows, int32_t cols, void* stream);

/*
 * pda_attention_prelude -- the prelude described above.
 *   x             bf16 [batch, hidden], 16-byte aligned.
 *   w_packed      packed bf16 [N, hidden] (pda_pack_weights), 16-byte aligned.
 *   bias          bf16 [N] or NULL.
 *   q_norm, k_norm  bf16 [head_dim] each, or both NULL (no norm).
 *   context_lens  int32 [batch] on the device (positions, see above).
 *   q_out         bf16 [batch, Hq, D]; k_out, v_out bf16 [batch, Hkv, D];
 *                 16-byte aligned.
 * Uses the (device, stream) workspace of paged_decode_attention for the fp32
 * projection (grown on demand; pda_prelude_workspace_reserve before graph
 * capture).  Asynchronous.  Errors: PDA_ERR_NULL, PDA_ERR_SHAPE,
 * PDA_ERR_UNSUPPORTED (dims outside the ranges above), PDA_ERR_ALIGN,
 * PDA_ERR_SCALE (theta or eps not finite / out of range), PDA_ERR_HIP.
 */
int pda_attention_prelude(const void* x, const void* w_packed, const void* bias, const void* q_norm,
                          const void* k_norm, const int32_t* context_lens, void* q_out, void* k_out,
                          void* v_out, const pda_prelude_dims* dims, void* stream);

/*
 * pda_attention_prelude_append -- the prelude with the KV append fused in:
 * k and v of sequence b are written (bf16) straight into the paged caches at
 * position context_lens[b] - 1, as pda_kv_append would, and q to q_out.
 * k_cache, v_cache, block_table, page_size, num_pages and max_pages_per_seq
 * as for paged_decode_attention (caches written in place, only those slots);
 * sequences with length 0 append nothing.  Other arguments and errors as
 * for pda_attention_prelude.
 */
int pda_attention_prelude_append(const void* x, const void* w_packed, const void* bias,
                                 const void* q_norm, const void* k_norm, const int32_t* context_lens,
                                 void* q_out, void* k_cache, void* v_cache, const int32_t* block_table,
                                 int32_t page_size, int32_t num_pages, int32_t max_pages_per_seq,
                                 const pda_prelude_dims* dims, void* stream);

/* [library interface] Grow the (current device, stream) workspace for a
   prelude of these dims. */
int pda_prelude_workspace_reserve(const pda_prelude_dims* dims, void* stream);

/*
 * ---------------------------------------------------------------------------
 * pda_o_proj_residual_norm -- the step after attention, the paper's kernel
 * family (v) (Method, "Principle-Driven LLM Kernel Generator": the output
 * projection fused with the residual add and the RMSNorm that follows):
 *
 *   z = W_o a + residual          (the new residual stream)
 *   h = z / sqrt(mean(z^2) + eps) * norm_w   (over the hidden features)
 *
 *   attn          bf16 [batch, in_features] (the heads' outputs concatenated),
 *                 16-byte aligned.
 *   w_packed      W_o bf16 [hidden, in_features], packed by pda_pack_weights.
 *   residual      bf16 [batch, hidden]; norm_w bf16 [hidden].
 *   residual_out  bf16 [batch, hidden]: z rounded once (may be residual itself,
 *                 updated in place); normed_out bf16 [batch, hidden]: h, from
 *                 the unrounded z; must not be residual_out.
 *   batch 0..256 (above 64, hidden a multiple of 128); in_features a
 *   multiple of 32 up to 65536; hidden a multiple of 16 up to 32768; eps
 *   finite and >= 0.
 * Uses the (device, stream) workspace (pda_o_proj_workspace_reserve before
 * graph capture).  Asynchronous.  Errors as for pda_attention_prelude.
 * ---------------------------------------------------------------------------
 */
int pda_o_proj_residual_norm(const void* attn, const void* w_packed, const void* residual, const void* norm_w,
                             void* residual_out, void* normed_out, int32_t batch, int32_t in_features,
                             int32_t hidden, float eps, void* stream);
/* [library interface] Grow the (current device, stream) workspace for an
   o_proj call of this shape. */
int pda_o_proj_workspace_reserve(int32_t batch, int32_t in_features, int32_t hidden, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* PDA_H */
