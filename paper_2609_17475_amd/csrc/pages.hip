// Page-run copies between one layer's pool and a packed buffer, for prefix
// snapshots and their restoration (Sec. 3.4, "Keep Checkpointing from
// Undoing the Savings"; Appendix A, Fig. kv-detail (b)): a snapshot reads the
// request's pages where they are (views of the live pool, no device-side copy
// of the cache) and restoration writes the packed runs back into pages of the
// existing pool.
//
// The pool keeps each page's bytes for all KV heads together: K codes
// [Hkv][P][d/2], K (scale, bias) words [Hkv][P][d/G], and the same for V.  A
// packed page is those four runs in that order (page_bytes =
// 2 Hkv P (d/2 + 4 d/G)), so packing page table[first + i] writes bytes
// [i page_bytes, (i + 1) page_bytes) of the buffer, which is device memory
// (the snapshot writer moves it to the host by copies).  A page ID outside
// the pool packs as zeros and is skipped on unpacking.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "jfkv.h"
#include "jfkv_internal.h"

namespace {

constexpr int kThreads = 256;
constexpr int kVecs = 4;  // 16-byte words per thread, their loads issued together

// UNPACK = false: pool -> buffer; true: buffer -> pool.
template <bool UNPACK>
__global__ __launch_bounds__(kThreads) void page_runs_kernel(
    uint4* __restrict__ k_codes, uint4* __restrict__ k_meta, uint4* __restrict__ v_codes,
    uint4* __restrict__ v_meta, const int32_t* __restrict__ table, int first, int NP,
    uint32_t codes16, uint32_t meta16, uint4* __restrict__ buf) {
  const int i = blockIdx.y;  // page of the range
  const int32_t page = table[first + i];
  const bool ok = (unsigned)page < (unsigned)NP;
  const uint32_t page16 = 2 * (codes16 + meta16);
  uint4* pb = buf + (size_t)i * page16;
  const uint32_t base = blockIdx.x * (kThreads * kVecs) + threadIdx.x;
  uint4 x[kVecs];
  uint4* at[kVecs];  // the word's place in the pool (null: past the page or not in the pool)
#pragma unroll
  for (int v = 0; v < kVecs; ++v) {
    const uint32_t o = base + v * kThreads;
    uint4* p = nullptr;
    if (ok && o < page16) {
      uint32_t r = o;
      if (r < codes16) {
        p = k_codes + (size_t)page * codes16 + r;
      } else if ((r -= codes16) < meta16) {
        p = k_meta + (size_t)page * meta16 + r;
      } else if ((r -= meta16) < codes16) {
        p = v_codes + (size_t)page * codes16 + r;
      } else {
        r -= codes16;
        p = v_meta + (size_t)page * meta16 + r;
      }
    }
    at[v] = p;
    if constexpr (UNPACK) {
      if (p) x[v] = pb[o];
    } else {
      x[v] = p ? *p : make_uint4(0u, 0u, 0u, 0u);
    }
  }
#pragma unroll
  for (int v = 0; v < kVecs; ++v) {
    const uint32_t o = base + v * kThreads;
    if constexpr (UNPACK) {
      if (at[v]) *at[v] = x[v];
    } else {
      if (o < page16) pb[o] = x[v];
    }
  }
}

}  // namespace

namespace jfkv {

size_t page_bytes(const jf_kv_layout& L) {
  return 2 * ((size_t)L.num_kv_heads * L.page_size *
              ((size_t)L.head_dim / 2 + 4 * (size_t)(L.head_dim / L.group_size)));
}

hipError_t launch_page_runs(const jf_kv_layout& L, const jf_kv_pool_ptrs& pool,
                            const int32_t* block_table, int32_t first, int32_t count, void* buf,
                            bool unpack, hipStream_t stream) {
  if (count == 0) return hipSuccess;
  const size_t codes = (size_t)L.num_kv_heads * L.page_size * (L.head_dim / 2);
  const size_t meta = (size_t)L.num_kv_heads * L.page_size * (L.head_dim / L.group_size) * 4;
  const uint32_t codes16 = (uint32_t)(codes / 16), meta16 = (uint32_t)(meta / 16);
  const uint32_t page16 = 2 * (codes16 + meta16);
  dim3 grid((page16 + kThreads * kVecs - 1) / (kThreads * kVecs), (unsigned)count);
  auto args = [&](auto kern) {
    hipLaunchKernelGGL(kern, grid, dim3(kThreads), 0, stream, static_cast<uint4*>(pool.k_codes),
                       static_cast<uint4*>(pool.k_meta), static_cast<uint4*>(pool.v_codes),
                       static_cast<uint4*>(pool.v_meta), block_table, first, L.num_pages,
                       codes16, meta16, static_cast<uint4*>(buf));
  };
  if (unpack)
    args(page_runs_kernel<true>);
  else
    args(page_runs_kernel<false>);
  return hipGetLastError();
}

}  // namespace jfkv
