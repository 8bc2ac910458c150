// KV append for MI355X (gfx950): the step before decode attention in the
// paper's decode loop (Method, "Kernel Customization and Multi-Request
// Adaptation": a small scatter kernel writes the step's new key and value
// vectors into the paged cache, and attention then runs with the sequence
// length advanced by one).
//
// The length already counts the new token, so sequence b's vectors land at
// position L_b - 1: page block_table[b, (L_b-1) / P], slot (L_b-1) % P, every
// kv head.  With T new tokens per sequence (a chunk of prefill, or several
// draft tokens) the length counts all T and token j lands at L_b - T + j;
// positions below 0 write nothing.  Pure data movement of 4*Hkv*D bytes per sequence (read and
// write), far below anything HBM-bound: the kernel is one launch of one
// thread per 16-byte chunk, so each (sequence, kv head) row of D bf16 is
// moved by D/8 consecutive lanes with 16-byte accesses.
//
// Page ids and lengths read from device memory are clamped into range (a
// length into [0, maxp*P], a page id into [0, num_pages)), so bad device
// contents cannot address outside the pool.
#include "pda_append.h"

namespace pda {
namespace {

typedef unsigned u32x4 __attribute__((ext_vector_type(4)));

template <int D>
__global__ __launch_bounds__(kAppendThreads) void append_kernel(
    const uint16_t* __restrict__ k_new, const uint16_t* __restrict__ v_new, uint16_t* __restrict__ kc,
    uint16_t* __restrict__ vc, const int32_t* __restrict__ bt, const int32_t* __restrict__ lens, int batch,
    int tokens, int hkv, int page_shift, int num_pages, int maxp) {
  constexpr int kChunks = D / 8;                    // 16-byte chunks per row
  const int64_t per_tok = 2 * static_cast<int64_t>(hkv) * kChunks;
  const int64_t i = static_cast<int64_t>(blockIdx.x) * kAppendThreads + threadIdx.x;
  if (i >= static_cast<int64_t>(batch) * tokens * per_tok) return;
  const int64_t bj = i / per_tok;                   // (sequence, new token)
  const int b = static_cast<int>(bj / tokens);
  const int j = static_cast<int>(bj - static_cast<int64_t>(b) * tokens);
  const int r = static_cast<int>(i - bj * per_tok);  // (K|V, kv head, chunk)
  const int which = r / (hkv * kChunks);
  const int g = (r / kChunks) % hkv;
  const int chunk = r % kChunks;

  const int max_ctx = maxp << page_shift;
  int L = lens[b];
  L = L < 0 ? 0 : (L > max_ctx ? max_ctx : L);
  const int t = L - tokens + j;                     // this token's position
  if (t < 0) return;
  const unsigned raw = static_cast<unsigned>(bt[static_cast<int64_t>(b) * maxp + (t >> page_shift)]);
  const int64_t page = raw < static_cast<unsigned>(num_pages) ? raw : num_pages - 1;
  const int slot = t & ((1 << page_shift) - 1);

  const int64_t dst = (((page << page_shift) + slot) * hkv + g) * D + 8 * chunk;
  const int64_t src = (bj * hkv + g) * D + 8 * chunk;
  const uint16_t* from = which ? v_new : k_new;
  uint16_t* to = which ? vc : kc;
  *reinterpret_cast<u32x4*>(to + dst) = *reinterpret_cast<const u32x4*>(from + src);
}

}  // namespace

hipError_t launch_append_kernel(const AppendArgs& a, hipStream_t st) {
  const int64_t n = static_cast<int64_t>(a.batch) * a.tokens * 2 * a.hkv * (a.head_dim / 8);
  const dim3 grid(static_cast<unsigned>((n + kAppendThreads - 1) / kAppendThreads));
  if (a.head_dim == 128)
    hipLaunchKernelGGL((append_kernel<128>), grid, dim3(kAppendThreads), 0, st, a.k_new, a.v_new, a.k, a.v,
                       a.bt, a.lens, a.batch, a.tokens, a.hkv, a.page_shift, a.num_pages, a.maxp);
  else if (a.head_dim == 256)
    hipLaunchKernelGGL((append_kernel<256>), grid, dim3(kAppendThreads), 0, st, a.k_new, a.v_new, a.k, a.v,
                       a.bt, a.lens, a.batch, a.tokens, a.hkv, a.page_shift, a.num_pages, a.maxp);
  else
    hipLaunchKernelGGL((append_kernel<64>), grid, dim3(kAppendThreads), 0, st, a.k_new, a.v_new, a.k, a.v,
                       a.bt, a.lens, a.batch, a.tokens, a.hkv, a.page_shift, a.num_pages, a.maxp);
  return hipGetLastError();
}

}  // namespace pda
