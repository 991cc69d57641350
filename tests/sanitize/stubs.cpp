// CPU stand-ins for the HIP runtime calls and kernel launchers that the host
// side of libjfkv.so (csrc/jfkv_host.cpp) uses, so that it can be built and
// exercised under AddressSanitizer and UndefinedBehaviorSanitizer on a
// machine without a GPU.  Test infrastructure only.
//
// Memory kinds: the driver registers the ranges it treats as device memory
// and as pinned host memory; hipPointerGetAttributes answers from that
// registry.  Copies run synchronously.  The page-run launcher performs the
// copy on the CPU (pool arrays are host memory here); the other launchers do
// nothing and report success, since their device work is not what this build
// checks.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstring>
#include <vector>

#include "jfkv_internal.h"

namespace {
struct Range {
  const char* p;
  size_t n;
  hipMemoryType kind;
};
std::vector<Range>& ranges() {
  static std::vector<Range> r;
  return r;
}
thread_local hipError_t g_last = hipSuccess;
}  // namespace

void stub_register(const void* p, size_t n, bool device) {
  ranges().push_back({static_cast<const char*>(p), n, device ? hipMemoryTypeDevice : hipMemoryTypeHost});
}

void stub_clear() { ranges().clear(); }

extern "C" {

hipError_t hipPointerGetAttributes(hipPointerAttribute_t* a, const void* p) {
  const char* c = static_cast<const char*>(p);
  for (const Range& r : ranges())
    if (c >= r.p && c < r.p + r.n) {
      std::memset(a, 0, sizeof(*a));
      a->type = r.kind;
      return hipSuccess;
    }
  g_last = hipErrorInvalidValue;
  return hipErrorInvalidValue;
}

hipError_t hipGetLastError(void) {
  hipError_t e = g_last;
  g_last = hipSuccess;
  return e;
}

const char* hipGetErrorString(hipError_t e) { return e == hipSuccess ? "no error" : "stub error"; }

hipError_t hipEventCreateWithFlags(hipEvent_t* e, unsigned) {
  *e = reinterpret_cast<hipEvent_t>(new int(0));
  return hipSuccess;
}

hipError_t hipEventDestroy(hipEvent_t e) {
  delete reinterpret_cast<int*>(e);
  return hipSuccess;
}

hipError_t hipEventRecord(hipEvent_t, hipStream_t) { return hipSuccess; }
hipError_t hipEventSynchronize(hipEvent_t) { return hipSuccess; }
hipError_t hipStreamSynchronize(hipStream_t) { return hipSuccess; }

hipError_t hipMemcpyAsync(void* dst, const void* src, size_t n, hipMemcpyKind, hipStream_t) {
  std::memcpy(dst, src, n);
  return hipSuccess;
}

}  // extern "C"

namespace jfkv {

size_t page_bytes(const jf_kv_layout& L) {
  return 2 * ((size_t)L.num_kv_heads * L.page_size *
              ((size_t)L.head_dim / 2 + 4 * (size_t)(L.head_dim / L.group_size)));
}

// The page-run copy on the CPU: page table[first + i] <-> bytes
// [i page_bytes, (i + 1) page_bytes) of buf, as K codes, K meta, V codes,
// V meta runs; pages outside the pool pack as zeros and are skipped when
// unpacking.
hipError_t launch_page_runs(const jf_kv_layout& L, const jf_kv_pool_ptrs& pool,
                            const int32_t* table, int32_t first, int32_t count, void* buf,
                            bool unpack, hipStream_t) {
  const size_t codes = (size_t)L.num_kv_heads * L.page_size * (L.head_dim / 2);
  const size_t meta = (size_t)L.num_kv_heads * L.page_size * (L.head_dim / L.group_size) * 4;
  char* runs[4] = {static_cast<char*>(pool.k_codes), static_cast<char*>(pool.k_meta),
                   static_cast<char*>(pool.v_codes), static_cast<char*>(pool.v_meta)};
  const size_t sizes[4] = {codes, meta, codes, meta};
  char* b = static_cast<char*>(buf);
  for (int32_t i = 0; i < count; ++i) {
    const int32_t page = table[first + i];
    const bool ok = page >= 0 && page < L.num_pages;
    for (int r = 0; r < 4; ++r) {
      char* pool_run = runs[r] + (size_t)(ok ? page : 0) * sizes[r];
      if (unpack) {
        if (ok) std::memcpy(pool_run, b, sizes[r]);
      } else if (ok) {
        std::memcpy(b, pool_run, sizes[r]);
      } else {
        std::memset(b, 0, sizes[r]);
      }
      b += sizes[r];
    }
  }
  return hipSuccess;
}

hipError_t launch_quantize_append(const jf_kv_layout&, const jf_kv_pool_ptrs&, const void*,
                                  const void*, const int32_t*, const int32_t*, const int32_t*,
                                  int32_t, int32_t, int32_t, hipStream_t) {
  return hipSuccess;
}
hipError_t launch_decode(const jf_kv_layout&, const jf_kv_pool_ptrs&, const void*, const void*,
                         const void*, int32_t, int32_t, const int32_t*, int32_t, const int32_t*,
                         float, int32_t, void*, void*, hipStream_t, int32_t) {
  return hipSuccess;
}
hipError_t launch_decode_static(const jf_kv_layout&, const jf_kv_pool_ptrs&, const void*,
                                const void*, const void*, int32_t, int32_t, const int32_t*,
                                int32_t, const int32_t*, float, int32_t, void*, hipStream_t) {
  return hipSuccess;
}
hipError_t launch_prefill(const jf_kv_layout&, const jf_kv_pool_ptrs&, const void*, const void*,
                          const void*, int32_t, int32_t, const int32_t*, int32_t, int32_t, float,
                          void*, hipStream_t) {
  return hipSuccess;
}
hipError_t launch_reconstruct(const jf_kv_layout&, const jf_kv_pool_ptrs&, const int32_t*,
                              int32_t, int32_t, int32_t, int32_t, void*, void*, hipStream_t) {
  return hipSuccess;
}
hipError_t launch_tq4_encode(const jf_kv_layout&, void*, void*, const void*, const float*,
                             const float*, const int32_t*, const int32_t*, const int32_t*,
                             int32_t, int32_t, int32_t, hipStream_t) {
  return hipSuccess;
}
hipError_t launch_tq4_decode(const jf_kv_layout&, const void*, const void*, const void*,
                             const void*, const float*, const float*, const float*, const void*,
                             int32_t, int32_t, const int32_t*, int32_t, const int32_t*, float,
                             int32_t, void*, void*, hipStream_t) {
  return hipSuccess;
}
hipError_t launch_tq4_reconstruct(const jf_kv_layout&, const void*, const void*, const void*,
                                  const void*, const float*, const float*, const float*,
                                  const int32_t*, int32_t, int32_t, int32_t, void*, void*,
                                  hipStream_t) {
  return hipSuccess;
}
hipError_t launch_read_stream(const void*, size_t, int32_t, uint32_t*, hipStream_t) {
  return hipSuccess;
}

}  // namespace jfkv
