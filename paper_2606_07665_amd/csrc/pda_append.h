// Internal interface of the KV append kernel (not part of the public ABI).
#pragma once
#include <hip/hip_runtime.h>
#include <cstdint>

namespace pda {

constexpr int kAppendThreads = 256;

struct AppendArgs {
  const uint16_t* k_new;  // bf16 [batch, tokens, hkv, head_dim]
  const uint16_t* v_new;
  uint16_t* k;            // bf16 [num_pages, page_size, hkv, head_dim], written in place
  uint16_t* v;
  const int32_t* bt;      // [batch, maxp]
  const int32_t* lens;    // [batch], counting the new token
  int batch, tokens, hkv, head_dim, page_shift, num_pages, maxp;
};

hipError_t launch_append_kernel(const AppendArgs& a, hipStream_t st);

}  // namespace pda
