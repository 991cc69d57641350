// Internal declarations shared by the host dispatcher and the kernel files
// of libjfkv.so.  Not part of the public ABI (include/jfkv.h is).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "jfkv.h"

namespace jfkv {

// Decode workspace: a fixed region of uint32 completion counters (one per
// request, KV head and head chunk; room for B * Hq <= kDecodeMaxHeads), then
// the fp32 split records [B][Hq][max_splits][d + 4] (o/l, m, l; 16-byte
// aligned records).  The fixed
// size keeps the counters where no call's records can land.
constexpr int32_t kDecodeMaxHeads = 65536;
constexpr size_t kDecodeCounterBytes = (size_t)kDecodeMaxHeads * sizeof(uint32_t);
inline size_t decode_workspace_bytes(int32_t B, int32_t Hq, int32_t head_dim, int32_t max_splits) {
  return kDecodeCounterBytes + (size_t)B * Hq * max_splits * (head_dim + 4) * sizeof(float);
}

// Allocation-free decode step: a device array of kStaticScratchBytes per
// device, its first kStaticTicketBytes completion counters (room for
// B * Hkv * ceil(Gq / 4) <= kStaticTickets), then split records
// [B][Hq][max_splits][d + 4] fp32.
constexpr size_t kStaticScratchBytes = (size_t)8 << 20;
constexpr size_t kStaticTicketBytes = 65536;
constexpr int64_t kStaticTickets = (int64_t)(kStaticTicketBytes / sizeof(uint32_t));

// Compute units of the current device (queried once per device).
int num_cus();

// Geometry accepted by every device entry point (validated on the host).
bool geometry_supported(const jf_kv_layout& L);

// Kernel launchers.  They assume validated arguments and return the HIP
// launch status.
hipError_t launch_quantize_append(const jf_kv_layout& L, const jf_kv_pool_ptrs& pool,
                                  const void* k_new, const void* v_new,
                                  const int32_t* cu_tok, const int32_t* start_pos,
                                  const int32_t* block_tables, int32_t B,
                                  int32_t max_pages, int32_t total_tok,
                                  hipStream_t stream);

// k_new/v_new non-null: the fused decode step (append one row per request
// at position seq_lens[b] - 1, then attend).  sq > 1 (k_new null): the
// short verifier, num_q_heads = query heads * sq (q and out token-major).
hipError_t launch_decode(const jf_kv_layout& L, const jf_kv_pool_ptrs& pool,
                         const void* k_new, const void* v_new,
                         const void* q, int32_t B, int32_t num_q_heads,
                         const int32_t* block_tables, int32_t max_pages,
                         const int32_t* seq_lens, float softmax_scale,
                         int32_t max_splits, void* workspace, void* out,
                         hipStream_t stream, int32_t sq = 1);

// The same step with its counters and records in the library's static
// device array (the caller passes no workspace).
hipError_t launch_decode_static(const jf_kv_layout& L, const jf_kv_pool_ptrs& pool,
                                const void* k_new, const void* v_new, const void* q, int32_t B,
                                int32_t num_q_heads, const int32_t* block_tables,
                                int32_t max_pages, const int32_t* seq_lens, float softmax_scale,
                                int32_t max_splits, void* out, hipStream_t stream);

// Page -> operand reconstruction of KV heads kv0 .. kv0 + num_heads - 1 at
// positions 0 .. n_pos - 1 of one request: fp16 [num_heads][n_pos][d] K and V.
hipError_t launch_reconstruct(const jf_kv_layout& L, const jf_kv_pool_ptrs& pool,
                              const int32_t* block_table, int32_t max_pages, int32_t n_pos,
                              int32_t kv0, int32_t num_heads, void* k_out, void* v_out,
                              hipStream_t stream);
hipError_t launch_tq4_reconstruct(const jf_kv_layout& L, const void* k_words, const void* k_norms,
                                  const void* v_words, const void* v_norms, const float* k_signs,
                                  const float* v_signs, const float* centroids,
                                  const int32_t* block_table, int32_t n_pos, int32_t kv0,
                                  int32_t num_heads, void* k_out, void* v_out,
                                  hipStream_t stream);

// Packed bytes of one page (all KV heads: K codes, K meta, V codes, V meta),
// and the page-run copy kernel (unpack: buffer -> pool).
size_t page_bytes(const jf_kv_layout& L);
hipError_t launch_page_runs(const jf_kv_layout& L, const jf_kv_pool_ptrs& pool,
                            const int32_t* block_table, int32_t first, int32_t count, void* buf,
                            bool unpack, hipStream_t stream);

hipError_t launch_prefill(const jf_kv_layout& L, const jf_kv_pool_ptrs& pool,
                          const void* q, const void* k_chunk, const void* v_chunk,
                          int32_t T, int32_t num_q_heads,
                          const int32_t* block_table, int32_t max_pages,
                          int32_t prefix_len, float softmax_scale, void* out,
                          hipStream_t stream);

hipError_t launch_tq4_encode(const jf_kv_layout& L, void* words, void* norms, const void* x,
                             const float* signs, const float* centroids, const int32_t* cu_tok,
                             const int32_t* start_pos, const int32_t* block_tables, int32_t B,
                             int32_t max_pages, int32_t total_tok, hipStream_t stream);

hipError_t launch_tq4_decode(const jf_kv_layout& L, const void* k_words, const void* k_norms,
                             const void* v_words, const void* v_norms, const float* k_signs,
                             const float* v_signs, const float* centroids, const void* q,
                             int32_t B, int32_t Hq, const int32_t* block_tables,
                             int32_t max_pages, const int32_t* seq_lens, float softmax_scale,
                             int32_t max_splits, void* ws, void* out, hipStream_t stream);

// Read-rate calibration: one pass over bytes (a multiple of 16) of buf.
hipError_t launch_read_stream(const void* buf, size_t bytes, int32_t blocks, uint32_t* sink,
                              hipStream_t stream);

}  // namespace jfkv
