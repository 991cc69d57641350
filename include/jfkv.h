/*
 * jfkv.h -- C ABI of libjfkv.so: attention executed directly over a
 * group-wise 4-bit quantized, paged KV cache on AMD Instinct MI355X (gfx950).
 *
 * The operations follow the KVExec component of "JustFit: Just-in-Time State
 * Management for Local LLM Serving":
 *   - a fixed backing pool of 256-token pages, a per-request page table that
 *     maps token order to pages, page IDs returned to a free list on
 *     completion (Background, "Compact histories need reusable storage");
 *   - reference-counted pages shared by requests with a common prefix and
 *     all-or-nothing page reservation (Sec. 3.3, eq. reservation and the
 *     refcounted shared prefixes it describes; Algorithm 1 recycles
 *     zero-reference pages after releasing a request);
 *   - single-query decode that reads the compressed pages directly, and
 *     prefill that consumes the same pages as floating operands (Sec. 3.1,
 *     "Decode and prefill need different kernels"); query heads grouped
 *     over shared KV heads, each head independent (eq. groupattention);
 *   - bounded temporary storage: the decode workspace has a size fixed by
 *     the caller's split cap, independent of context length (Sec. 3.1,
 *     "Finish one head group ..." motivates bounding workspace; eq.
 *     layerbytes is what the fused prefill avoids materializing).
 * Stored format: affine 4-bit codes with one fp16 scale and one fp16 bias
 * per group of head_dim elements (the affine 4-bit format the Introduction
 * describes for weights: a scale and an offset per group), eight codes per 32-bit word
 * (Appendix A, Table codec, per-vector storage).
 *
 * ---------------------------------------------------------------------
 * Pool byte layout (per layer; one set for K and one for V):
 *   k_codes  uint8 [NP][Hkv][P][d/2]          byte j of a position's row =
 *                                             code(2j) | code(2j+1) << 4
 *   v_codes  uint8 [NP][Hkv][P/2][d/4][2][2]  positions paired (2s, 2s+1):
 *                                             dims 4u..4u+3 of slot t are the
 *                                             2 bytes at ((t/2)*(d/4)+u)*4 +
 *                                             (t%2)*2, holding code(4u) |
 *                                             code(4u+1)<<4 and code(4u+2) |
 *                                             code(4u+3)<<4
 *   k_meta, v_meta  fp16 [NP][Hkv][P][d/G][2]  (scale, bias) per group
 * Bytes per position per layer: 2*Hkv*(d/2 + 4*d/G) (1,152 at Hkv=8,
 * d=128, G=64).
 *
 * Quantizer (bit-exact contract), per group x_0..x_{G-1} of fp16 values:
 *   mn, mx   = min, max (binary32; -0 orders below +0)
 *   bias     = fp16 of mn rounded toward -inf
 *   range    = mx - mn; step = range / 15  (binary32, IEEE round-to-nearest)
 *   scale    = fp16 of step rounded toward +inf; +0 when range == 0
 *   code_i   = 0 if scale == 0, else clamp(rint((x_i - bias) / scale), 0, 15)
 *              with the subtraction and division separate binary32 ops and
 *              rint rounding half to even
 *   x^_i     = scale * code_i + bias
 * Inputs must be finite.
 *
 * ---------------------------------------------------------------------
 * Conventions for every entry point:
 *   - Every function returns jf_status; no C++ exception crosses the ABI.
 *   - Arguments are validated before anything is launched; a call that
 *     fails validation has no side effect.  jf_last_error() then returns a
 *     message (thread-local; valid until the next jf_* call on the thread).
 *   - Device pointers are caller-owned (allocated by the caller, e.g. by
 *     PyTorch); the library never allocates or frees device memory.  Device
 *     work is enqueued asynchronously on the given stream (NULL = the
 *     default stream); faults inside kernels surface at the caller's next
 *     synchronization.  A launch failure returns JF_ERR_DEVICE.
 *   - Host page-pool objects are owned by the library from _create until
 *     _destroy and are not thread-safe: callers serialize calls per pool.
 *   - GQA mapping: query head h reads KV head h / (num_q_heads / Hkv).
 */
#ifndef JFKV_H
#define JFKV_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  JF_OK = 0,
  JF_ERR_INVALID = 1,     /* bad argument (NULL, shape, range)               */
  JF_ERR_NO_PAGES = 2,    /* page reservation could not be satisfied         */
  JF_ERR_DEVICE = 3,      /* HIP launch or runtime error                     */
  JF_ERR_UNSUPPORTED = 4, /* valid but not implemented geometry              */
  JF_ERR_STATE = 5,       /* operation not allowed in the object's state     */
  JF_ERR_IO = 6           /* host file I/O failed (snapshots)                */
} jf_status;

/* Message for the last failing jf_* call on this thread ("" if none). */
const char* jf_last_error(void);

/* Library version string. */
const char* jf_version(void);

/* Pool geometry.  Supported: page_size a multiple of 64 (256 in the paper's
 * geometry); head_dim 64, 128 or 256; group_size 32, 64 or 128 dividing
 * head_dim; num_kv_heads >= 1; num_pages >= 1. */
typedef struct {
  int32_t page_size;
  int32_t num_kv_heads;
  int32_t head_dim;
  int32_t group_size;
  int32_t num_pages;
} jf_kv_layout;

/* Device pointers to one layer's pools (layout above). */
typedef struct {
  void* k_codes;
  void* k_meta;
  void* v_codes;
  void* v_meta;
} jf_kv_pool_ptrs;

/* Bytes of one codes array and of one meta array for the layout (the same
 * for K and V).  Errors: JF_ERR_INVALID / JF_ERR_UNSUPPORTED for bad
 * geometry or NULL outputs. */
jf_status jf_kv_pool_bytes(const jf_kv_layout* layout, size_t* codes_bytes,
                           size_t* meta_bytes);

/* ---------------------------------------------------------------------
 * Host page allocator and per-request page tables (paging: Background,
 * "Compact histories need reusable storage"; shared prefixes and
 * reservation: eq. reservation; recycling: Algorithm 1).
 * ------------------------------------------------------------------- */
typedef struct jf_page_pool jf_page_pool;

/* Create a pool of num_pages page IDs.  The free list is a stack; with
 * shuffle_seed != 0 its initial order is a seeded permutation (so
 * consecutive reservations receive non-contiguous physical pages), with 0
 * pages are handed out in increasing order.  *out receives the pool. */
jf_status jf_page_table_pool_create(int32_t num_pages, int32_t page_size,
                                    uint64_t shuffle_seed, jf_page_pool** out);
jf_status jf_page_table_pool_destroy(jf_page_pool* pool);

/* New empty request (length 0, no pages); *seq receives its handle. */
jf_status jf_page_table_create(jf_page_pool* pool, int32_t* seq);

/* New request that shares (copy-free, reference count + 1) the first
 * prefix_len positions of src.  prefix_len must be a multiple of page_size
 * and at most src's length, so the new request's next write lands on a page
 * of its own.  Its length starts at prefix_len. */
jf_status jf_page_table_fork(jf_page_pool* pool, int32_t src,
                             int32_t prefix_len, int32_t* seq);

/* Append the n given free pages to seq's page list (explicit placement,
 * e.g. a reversed or shuffled mapping).  JF_ERR_STATE if any is not free
 * or listed twice; nothing changes then. */
jf_status jf_page_table_assign(jf_page_pool* pool, int32_t seq,
                               const int32_t* page_ids, int32_t n);

/* Ensure seq owns ceil(new_len / page_size) pages, taking missing ones from
 * the free list; all or nothing (JF_ERR_NO_PAGES leaves seq unchanged).
 * JF_ERR_STATE if positions length..new_len-1 would fall on a page whose
 * reference count is above one (shared pages are read-only). */
jf_status jf_page_table_reserve(jf_page_pool* pool, int32_t seq,
                                int32_t new_len);

/* Commit seq's length after its rows were appended; len must not exceed
 * its page capacity. */
jf_status jf_page_table_set_length(jf_page_pool* pool, int32_t seq,
                                   int32_t len);

/* Drop seq: each of its pages loses one reference; pages reaching zero go
 * back on the free list (last released, first reused).  The handle becomes
 * invalid (JF_ERR_STATE on reuse). */
jf_status jf_page_table_release(jf_page_pool* pool, int32_t seq);

/* Write the page tables of n requests as a host block table
 * [n][max_pages] (unused entries -1) and their lengths [n].  JF_ERR_INVALID
 * if a request has more than max_pages pages. */
jf_status jf_page_table_export(const jf_page_pool* pool, const int32_t* seqs,
                               int32_t n, int32_t max_pages,
                               int32_t* block_table, int32_t* lens);

/* Pages currently free, in use (reference count > 0), and the most pages
 * ever in use at once. */
jf_status jf_page_table_stats(const jf_page_pool* pool, int32_t* free_pages,
                              int32_t* used_pages, int32_t* high_water);

/* Number of pages of seq and its committed length. */
jf_status jf_page_table_info(const jf_page_pool* pool, int32_t seq,
                             int32_t* n_pages, int32_t* length);

/* ---------------------------------------------------------------------
 * Device work.
 * ------------------------------------------------------------------- */

/* Quantize rows of new K and V and write them into their pages (the
 * "pending cache writes" a step finishes before its pages may be released,
 * Algorithm 1).
 *   k_new, v_new  fp16 [total_tok][Hkv][d] (device), rows of all requests
 *                 concatenated;
 *   cu_tok        int32 [B+1] (device) row offsets: request b owns rows
 *                 cu_tok[b] .. cu_tok[b+1]-1, total_tok == cu_tok[B];
 *   start_pos     int32 [B] (device) logical position of each request's
 *                 first new row;
 *   block_tables  int32 [B][max_pages] (device) physical page of each
 *                 logical page.
 * Rows whose logical page is beyond max_pages or whose page ID is outside
 * [0, num_pages) are skipped (nothing is written for them).  The pages must
 * have been reserved and not be shared.  Codes, scales and biases are
 * bit-exact with the quantizer contract above. */
jf_status jf_kv_quantize_append(const jf_kv_layout* layout,
                                const jf_kv_pool_ptrs* pool,
                                const void* k_new, const void* v_new,
                                const int32_t* cu_tok,
                                const int32_t* start_pos,
                                const int32_t* block_tables, int32_t B,
                                int32_t max_pages, int32_t total_tok,
                                hipStream_t stream);

/* Workspace bytes jf_decode_attn_q4 needs: a fixed 262,144-byte region of
 * completion counters (room for B * num_q_heads <= 65,536; larger products
 * return JF_ERR_UNSUPPORTED), then B * num_q_heads * max_splits *
 * (head_dim + 4) * 4 bytes of fp32 partials (o/l, m, l per split, padded to
 * 16-byte records).  It does
 * not depend on sequence lengths. */
jf_status jf_decode_workspace_bytes(int32_t B, int32_t num_q_heads,
                                    int32_t head_dim, int32_t max_splits,
                                    size_t* bytes);

/* Single-query decode attention over the paged 4-bit cache: split-K
 * partials, then a log-sum-exp combine done by the last split of each
 * (request, KV head) to finish; one kernel on `stream`.
 *   q            fp16 [B][num_q_heads][d] (device)
 *   block_tables int32 [B][max_pages] (device)
 *   seq_lens     int32 [B] (device): request b attends to its logical
 *                positions 0..seq_lens[b]-1 (append first, then attend);
 *                values above max_pages*page_size are clamped; a request
 *                with length <= 0 gets an all-zero output row
 *   softmax_scale  logits = softmax_scale * q . k
 *   max_splits   cap on partials per request and KV head (1..1024); a
 *                request with n pages uses S = min(max_splits, n,
 *                max(1, floor(compute units / (num_kv_heads *
 *                ceil(Gq / H))))), H the query heads one block serves:
 *                h = 4 for 32-dim groups or head_dim 256, else 8, and
 *                H = 2h when Gq > h and head_dim <= 128, else h
 *                page-aligned splits of equal page counts, the remainder on
 *                the first (S depends on neither the batch nor the other
 *                requests, so a request's output is the same in any batch)
 *   workspace    device scratch of at least jf_decode_workspace_bytes().
 *                Its first 262,144 bytes (completion counters) must be zero
 *                before the first call, e.g. by allocating it zero-filled;
 *                every call that completes leaves them zero, so the same
 *                workspace serves any later call of any shape that fits.
 *                Calls that may overlap in time must not share one.
 *   out          fp16 [B][num_q_heads][d] (device)
 * Page IDs outside [0, num_pages) are never dereferenced; the positions
 * they would hold do not contribute. */
jf_status jf_decode_attn_q4(const jf_kv_layout* layout,
                            const jf_kv_pool_ptrs* pool, const void* q,
                            int32_t B, int32_t num_q_heads,
                            const int32_t* block_tables, int32_t max_pages,
                            const int32_t* seq_lens, float softmax_scale,
                            int32_t max_splits, void* workspace,
                            size_t workspace_bytes, void* out,
                            hipStream_t stream);

/* Short packed verification (Sec. 3.1, the speculative-verification
 * paragraph after eq. groupattention; Appendix A, "Codec and Attention
 * Dispatch": causal string masks, 2 to 4 queries).  The last num_queries
 * positions of request b (already appended: positions seq_lens[b] -
 * num_queries .. seq_lens[b] - 1) are its query tokens; token k sees the
 * positions 0 .. seq_lens[b] - num_queries + k (a causal mask aligned to the
 * end of the cache).  One page scan serves every token and query head of a
 * KV head chunk, as in jf_decode_attn_q4.
 *   q            fp16 [B][num_queries][num_q_heads][d] (device)
 *   num_queries  1..4 (1 is jf_decode_attn_q4); larger: JF_ERR_UNSUPPORTED
 *   workspace    at least jf_decode_workspace_bytes(B, num_q_heads *
 *                num_queries, d, max_splits); same zeroing rule as decode
 *   out          fp16 [B][num_queries][num_q_heads][d] (device)
 * Other arguments as jf_decode_attn_q4; a token whose visible length is
 * <= 0 gets an all-zero output row. */
jf_status jf_verify_attn_q4(const jf_kv_layout* layout,
                            const jf_kv_pool_ptrs* pool, const void* q,
                            int32_t B, int32_t num_queries, int32_t num_q_heads,
                            const int32_t* block_tables, int32_t max_pages,
                            const int32_t* seq_lens, float softmax_scale,
                            int32_t max_splits, void* workspace,
                            size_t workspace_bytes, void* out,
                            hipStream_t stream);

/* One decode step, append then attend, in one kernel: request b's new row
 * (k_new, v_new: fp16 [B][Hkv][d], device) is quantized into the pool at
 * logical position seq_lens[b] - 1 exactly as jf_kv_quantize_append would
 * write it (same codes, scales, biases and placement; a row whose position
 * is beyond max_pages * page_size or whose page ID is outside
 * [0, num_pages) is not written), and the query then attends to positions
 * 0..seq_lens[b]-1, the new row included, as in jf_decode_attn_q4 (same
 * arguments and workspace).  One launch per decode step instead of two
 * (append, then attend); the outputs and the pool are the same.  The row's
 * page must be reserved and not shared. */
jf_status jf_decode_step_q4(const jf_kv_layout* layout,
                            const jf_kv_pool_ptrs* pool, const void* k_new,
                            const void* v_new, const void* q, int32_t B,
                            int32_t num_q_heads, const int32_t* block_tables,
                            int32_t max_pages, const int32_t* seq_lens,
                            float softmax_scale, int32_t max_splits,
                            void* workspace, size_t workspace_bytes, void* out,
                            hipStream_t stream);

/* jf_decode_step_q4 without a workspace argument, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid allocation).  The step's completion counters and
 * split records live in a device array inside the library: 8 MiB per device
 * (64 KiB of counters, then records), held until the process ends; its
 * address is looked up once per device (hipGetSymbolAddress, which
 * allocates nothing), and the first call on a device also enqueues a small
 * kernel that zeroes the counters.  The call allocates and frees nothing.
 * Arguments, outputs and pool writes are those of jf_decode_step_q4 with the
 * same max_splits (the outputs are bitwise the same).
 * Limits: B * num_kv_heads * ceil(Gq / 4) <= 16,384 counters and
 * B * num_q_heads * max_splits * (head_dim + 4) * 4 <= 8,323,072 bytes of
 * records; larger requests return JF_ERR_INVALID (nothing launched).
 * Every call on a device shares that device's array and keeps its last
 * contents: calls that may overlap in time on one device (other streams,
 * other threads) race and must not be issued. */
jf_status jf_decode_step_q4_static(const jf_kv_layout* layout,
                                   const jf_kv_pool_ptrs* pool,
                                   const void* k_new, const void* v_new,
                                   const void* q, int32_t B,
                                   int32_t num_q_heads,
                                   const int32_t* block_tables,
                                   int32_t max_pages, const int32_t* seq_lens,
                                   float softmax_scale, int32_t max_splits,
                                   void* out, hipStream_t stream);

/* Chunked-prefill attention for one request: query i of the chunk sits at
 * absolute position prefix_len + i and attends to the dequantized prefix
 * positions 0..prefix_len-1 (through block_table) and, causally, to the
 * chunk's own fp16 rows 0..i.  The chunk is not written to the pool here:
 * call jf_kv_quantize_append afterwards.
 *   q        fp16 [T][num_q_heads][d] (device)
 *   k_chunk, v_chunk  fp16 [T][Hkv][d] (device)
 *   block_table  int32 [max_pages] (device); pages 0..ceil(prefix_len/P)-1
 *                are read; prefix_len must be <= max_pages * page_size
 *   out      fp16 [T][num_q_heads][d] (device)
 * Products run on fp16 matrix cores with fp32 accumulation.  Key codes
 * enter exactly, with scales and biases applied to the fp32 scores; prefix
 * values enter as (scale * code + bias) / 2 split into an fp16 high and low
 * part (exact to ~2^-21 relative, no fp16 overflow for any group), the
 * chunk's own fp16 rows exactly. */
jf_status jf_prefill_attn_q4(const jf_kv_layout* layout,
                             const jf_kv_pool_ptrs* pool, const void* q,
                             const void* k_chunk, const void* v_chunk,
                             int32_t T, int32_t num_q_heads,
                             const int32_t* block_table, int32_t max_pages,
                             int32_t prefix_len, float softmax_scale,
                             void* out, hipStream_t stream);

/* Page -> operand reconstruction of one head group for an SDPA-style
 * consumer (Background, "Stored format is not execution format", eq.
 * layerbytes; Sec. 3.1, "Finish one head group before starting the next",
 * eq. groupattention): the dequantized K and V vectors of KV heads
 * kv0 .. kv0 + num_heads - 1 at logical positions 0 .. n_pos - 1 of one
 * request, read through block_table, written as contiguous operands.  A
 * grouped prefill reconstructs one group (the paper's: two KV heads),
 * attends with that group's query heads, and reuses the same
 * 2 * num_heads * n_pos * d * 2 bytes for the next group.
 *   block_table  int32 [max_pages] (device); n_pos <= max_pages * page_size
 *   k_out, v_out fp16 [num_heads][n_pos][d] (device, 16-byte aligned,
 *                caller-owned); element = scale * code + bias rounded once to
 *                fp16 (nearest, ties to even: the exact value's rounding,
 *                not a rounding of an fp32 intermediate)
 * A page ID outside [0, num_pages) gives zero vectors.  n_pos = 0 launches
 * nothing. */
jf_status jf_reconstruct_q4(const jf_kv_layout* layout,
                            const jf_kv_pool_ptrs* pool,
                            const int32_t* block_table, int32_t max_pages,
                            int32_t n_pos, int32_t kv0, int32_t num_heads,
                            void* k_out, void* v_out, hipStream_t stream);

/* ------------------------------------------------------- snapshots
 * Prefix snapshots and their restoration (Sec. 3.4, "Keep Checkpointing
 * from Undoing the Savings"; Appendix A, Fig. kv-detail (b); Table writer).
 * A page of one layer's pool is packed as its four runs for all KV heads:
 * K codes, K (scale, bias), V codes, V (scale, bias), exactly as the pool
 * stores them (page_bytes = 2 * Hkv * page_size * (d/2 + 4 * d/G)). */

/* page_bytes of this layout. */
jf_status jf_kv_page_bytes(const jf_kv_layout* layout, size_t* bytes);

/* Pack pages block_table[first .. first+count-1] of one layer's pool, in
 * that order, into buf (count * page_bytes bytes of device memory, 16-byte
 * aligned); or unpack buf into those pages.  block_table: int32 (device).
 * A page ID outside [0, num_pages) packs as zeros and is skipped when
 * unpacking.  One kernel on stream; the pages are read (or written) where
 * they are.  A buf that is not device memory is rejected (JF_ERR_INVALID):
 * kernels never dereference host memory.  Pool codes 16-byte and meta
 * 4-byte aligned. */
jf_status jf_kv_pack_pages(const jf_kv_layout* layout, const jf_kv_pool_ptrs* pool,
                           const int32_t* block_table, int32_t first, int32_t count,
                           void* buf, hipStream_t stream);
jf_status jf_kv_unpack_pages(const jf_kv_layout* layout, const jf_kv_pool_ptrs* pool,
                             const int32_t* block_table, int32_t first, int32_t count,
                             const void* buf, hipStream_t stream);

/* Read-rate calibration (not part of the method): reads bytes (a positive
 * multiple of 16) of device memory at buf once, with the 16-byte
 * non-temporal loads of the HBM-bound kernels, `blocks` blocks of 512
 * threads each reading one contiguous share, and does nothing else.  The
 * time it takes on a buffer of the decode's size is the practical read
 * ceiling the kernels' fractions of peak are compared with.  sink: 4 bytes
 * of device memory (written only for a buffer whose words xor to a fixed
 * 96-bit pattern).  buf 16-byte aligned; blocks 1..65535.  One kernel on
 * stream. */
jf_status jf_calib_read_stream(const void* buf, size_t bytes, int32_t blocks, void* sink,
                               hipStream_t stream);

/* Save the first n_pos positions of one request, all n_layers layers
 * (pools[l]: the layers' pools, one layout), to a file in one pass.  The
 * pages are read in place through block_table (device; the same IDs in
 * block_table_host, checked to lie in the pool) and streamed to the host
 * through two caller buffers of staging_bytes each (at least two pages;
 * 16-byte aligned): staging_dev (device memory) and staging (pinned host
 * memory).  Each is used as two halves in turn: a kernel packs pages into a
 * device half, a copy moves them to the host half, and the host writes the
 * other half meanwhile, so the memory used is those buffers, whatever
 * n_pos is (no copy of the cache is made).  The file is written as
 * path + ".tmp" and renamed to path once complete and flushed (fsync), so
 * path holds either a whole snapshot or what it held before; on failure the
 * temporary file is removed.  Format: safetensors (8-byte little-endian
 * header length, JSON header, data), one U8 tensor "layer<l>" of shape
 * [ceil(n_pos / page_size)][page_bytes] per layer, the layout and n_pos in
 * the header's metadata; whole pages are saved (slots past n_pos as they
 * are).  Synchronous: returns once the file is published.  The request
 * keeps its pages, which must not change or be released until the call
 * returns.  JF_ERR_INVALID for staging buffers of the wrong kind; JF_ERR_IO
 * on file errors, with errno's text in jf_last_error. */
jf_status jf_snapshot_save(const char* path, const jf_kv_layout* layout,
                           const jf_kv_pool_ptrs* pools, int32_t n_layers,
                           const int32_t* block_table, const int32_t* block_table_host,
                           int32_t max_pages, int32_t n_pos, void* staging_dev,
                           void* staging, size_t staging_bytes, hipStream_t stream);

/* Restore a snapshot written by jf_snapshot_save with the same layout and
 * layer count into the pages of a request's table (block_table device,
 * block_table_host the same IDs; its first ceil(n_pos / page_size) entries
 * must be distinct pages of the pool, reserved by the caller), writing the
 * packed runs straight into those pages: pieces of the file are read into
 * the pinned staging halves in turn, copied to the device halves and
 * unpacked by a kernel while the next piece is read.  *n_pos_out receives
 * the snapshot's position count.  Synchronous.  JF_ERR_INVALID if the file
 * is not such a snapshot (header, layout, layer count or size differ), the
 * table is too short or lists a page twice, or a staging buffer is of the
 * wrong kind; JF_ERR_IO on read errors. */
jf_status jf_snapshot_restore(const char* path, const jf_kv_layout* layout,
                              const jf_kv_pool_ptrs* pools, int32_t n_layers,
                              const int32_t* block_table, const int32_t* block_table_host,
                              int32_t max_pages, void* staging_dev, void* staging,
                              size_t staging_bytes, int32_t* n_pos_out, hipStream_t stream);

/* ---------------------------------------------------------------- TQ4
 * The paper's own 4-bit format (Sec. 3.1, eq. codec; Appendix A, Table
 * codec): a 256-element vector x is stored as the fp16 norm of x and 256
 * 4-bit indices z, where z_i indexes the one of 16 shared centroids c
 * (ascending) nearest to coordinate i of the rotated unit vector
 * y = H_256 S x / (16 |x|) (H_256 the unnormalised Sylvester Hadamard matrix,
 * S = diag(signs)).  Reconstruction: x_hat = norm * S H_256 c[z] / 16.
 *
 * Pool (per layer, per K or V; caller-owned device memory), head-major
 * pages like the affine pool:
 *   words  u32  [num_pages][num_kv_heads][page_size][32]  element 8w + k of
 *               a vector in bits 4k..4k+3 of word w
 *   norms  fp16 [num_pages][num_kv_heads][page_size]
 * Only page_size, num_kv_heads, head_dim (256) and num_pages of the layout
 * are used; group_size is ignored. */
jf_status jf_tq4_pool_bytes(const jf_kv_layout* layout, size_t* words_bytes,
                            size_t* norms_bytes);

/* Encode-and-append total_tok rows of K or V (one call per tensor, each
 * with its own signs) into a TQ4 pool, async on `stream`, one kernel.
 *   x            fp16 [total_tok][num_kv_heads][256] (device, 8-byte aligned)
 *   signs        fp32 [256] (device, 16-byte aligned), each +1 or -1
 *   centroids    fp32 [16] (device), ascending
 *   cu_tok, start_pos, block_tables, B, max_pages: as in
 *                jf_kv_quantize_append (row i of request b goes to logical
 *                position start_pos[b] + i; rows whose position falls outside
 *                the table or whose page ID is outside [0, num_pages) are
 *                not written)
 * Norm: the float32 Euclidean norm, rounded to fp16 (+inf when the norm
 * exceeds the fp16 range, i.e. |x| >= 65520; such vectors are out of range
 * for decode).  Index of a coordinate:
 * the number of thresholds (c_j + c_{j+1}) / 2 (float32) it strictly exceeds.
 * A zero vector gets norm 0 and the indices of coordinate 0.
 * Errors: NULL or misaligned pointers, B or max_pages <= 0, total_tok < 0,
 * max_pages * page_size above INT32_MAX -> JF_ERR_INVALID; head_dim != 256
 * or total_tok * num_kv_heads above INT32_MAX -> JF_ERR_UNSUPPORTED; no
 * launch on error. */
jf_status jf_tq4_encode_append(const jf_kv_layout* layout, void* words,
                               void* norms, const void* x, const float* signs,
                               const float* centroids, const int32_t* cu_tok,
                               const int32_t* start_pos,
                               const int32_t* block_tables, int32_t B,
                               int32_t max_pages, int32_t total_tok,
                               hipStream_t stream);

/* Single-query decode attention over TQ4 pages (Sec. 3.1, eq. codec: the
 * page-native decode reads the packed indices and norms where they are
 * stored).  Query head h reads KV head h / (num_q_heads / Hkv); request b
 * attends to its logical positions 0..seq_lens[b]-1 through its page table.
 * Computed without reconstructing any vector: the query is rotated once
 * (q' = H S_k q / 16), each position's logit is softmax_scale * norm_k *
 * (q' . c[z_k]), the weighted sum u = sum_t p_t norm_v c[z_v] is kept in the
 * rotated space, and the output is S_v H u / (16 sum_t p_t).
 *   k_words, v_words  u32 [NP][Hkv][P][32] (TQ4 pool layout above), 16-byte
 *                     aligned; k_norms, v_norms fp16 [NP][Hkv][P], 16-byte
 *                     aligned
 *   k_signs, v_signs  fp32 [256] (device): the sign diagonals the vectors
 *                     were encoded with; centroids fp32 [16] (device)
 *   q, out            fp16 [B][num_q_heads][256] (device)
 *   block_tables, max_pages, seq_lens, softmax_scale, max_splits,
 *   workspace         as in jf_decode_attn_q4, the workspace sized by
 *                     jf_decode_workspace_bytes(B, num_q_heads, 256,
 *                     max_splits) (same zero-counter rules)
 * Arithmetic: centroids rounded to fp16 once, q' as an fp16 high plus low
 * part, products on fp16 matrix cores with fp32 accumulation.  A norm that
 * overflowed fp16 at encode time (|x| above 65504) is +inf and makes the
 * outputs of every query reading that position non-finite.
 * Errors: head_dim != 256, page_size not a multiple of 32 or more than 16
 * query heads per KV head -> JF_ERR_UNSUPPORTED; NULL or misaligned
 * pointers, bad sizes, a short workspace or a non-finite scale ->
 * JF_ERR_INVALID; no launch on error. */
jf_status jf_tq4_decode_attn(const jf_kv_layout* layout, const void* k_words,
                             const void* k_norms, const void* v_words,
                             const void* v_norms, const float* k_signs,
                             const float* v_signs, const float* centroids,
                             const void* q, int32_t B, int32_t num_q_heads,
                             const int32_t* block_tables, int32_t max_pages,
                             const int32_t* seq_lens, float softmax_scale,
                             int32_t max_splits, void* workspace,
                             size_t workspace_bytes, void* out,
                             hipStream_t stream);

/* TQ4 page -> operand reconstruction (Appendix A, Table codec: page lookup,
 * index unpacking, centroid lookup, inverse rotation and norm restoration
 * in one kernel; Sec. 3.1, eq. groupattention): x_hat = norm * S H_256
 * c[z] / 16 for KV heads kv0 .. kv0 + num_heads - 1 at logical positions
 * 0 .. n_pos - 1 of one request, as contiguous fp16 k_out, v_out
 * [num_heads][n_pos][256] (device, 8-byte aligned).  Arithmetic in fp32
 * (centroids as given, the transform's sums, then signs and norm / 16),
 * rounded once to fp16.  Pool, signs and centroids as in
 * jf_tq4_decode_attn; block_table int32 [max_pages] (device).  A page ID
 * outside [0, num_pages) gives zero vectors. */
jf_status jf_tq4_reconstruct(const jf_kv_layout* layout, const void* k_words,
                             const void* k_norms, const void* v_words,
                             const void* v_norms, const float* k_signs,
                             const float* v_signs, const float* centroids,
                             const int32_t* block_table, int32_t max_pages,
                             int32_t n_pos, int32_t kv0, int32_t num_heads,
                             void* k_out, void* v_out, hipStream_t stream);

#ifdef __cplusplus
}
#endif
#endif /* JFKV_H */
