// Host side of libjfkv.so: error reporting, argument validation, the page
// allocator with per-request page tables, and dispatch to the kernels.
//
// Paging follows the paper's Background paragraph "Compact histories need
// reusable storage" (fixed pool of 256-token pages, a page table per
// request, page IDs returned on completion); shared prefixes hold reference
// counts and reservation is all-or-nothing (Sec. 3.3, eq. reservation);
// releasing a request recycles its zero-reference pages (Algorithm 1).
#include <fcntl.h>
#include <sys/stat.h>
#include <unistd.h>

#include <algorithm>
#include <cerrno>
#include <climits>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <new>
#include <string>
#include <vector>

#include "jfkv_internal.h"

namespace {

thread_local std::string g_last_error;

jf_status fail(jf_status st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof(buf), fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return st;
}

jf_status ok() {
  g_last_error.clear();
  return JF_OK;
}

jf_status device_status(hipError_t e, const char* what) {
  if (e == hipSuccess) return ok();
  return fail(JF_ERR_DEVICE, "%s: %s", what, hipGetErrorString(e));
}

jf_status check_layout(const jf_kv_layout* L) {
  if (!L) return fail(JF_ERR_INVALID, "layout is NULL");
  if (L->page_size <= 0 || L->num_kv_heads <= 0 || L->head_dim <= 0 ||
      L->group_size <= 0 || L->num_pages <= 0)
    return fail(JF_ERR_INVALID, "layout fields must be positive");
  if (L->head_dim % L->group_size)
    return fail(JF_ERR_INVALID, "head_dim %d is not a multiple of group_size %d",
                L->head_dim, L->group_size);
  if (!jfkv::geometry_supported(*L))
    return fail(JF_ERR_UNSUPPORTED,
                "unsupported geometry (page_size %d must be a multiple of 64 and <= 4096, "
                "head_dim %d in {64,128,256}, group_size %d in {32,64,128})",
                L->page_size, L->head_dim, L->group_size);
  return JF_OK;
}

jf_status check_pool(const jf_kv_pool_ptrs* p) {
  if (!p || !p->k_codes || !p->k_meta || !p->v_codes || !p->v_meta)
    return fail(JF_ERR_INVALID, "pool pointers must be non-NULL");
  return JF_OK;
}

// splitmix64 (Steele, Lea, Flood 2014): a small seeded generator for the
// optional shuffled initial order of the free list.
uint64_t splitmix64(uint64_t& s) {
  uint64_t z = (s += 0x9e3779b97f4a7c15ull);
  z = (z ^ (z >> 30)) * 0xbf58476d1ce4e5b9ull;
  z = (z ^ (z >> 27)) * 0x94d049bb133111ebull;
  return z ^ (z >> 31);
}

}  // namespace

namespace jfkv {
bool geometry_supported(const jf_kv_layout& L) {
  bool d_ok = L.head_dim == 64 || L.head_dim == 128 || L.head_dim == 256;
  bool g_ok = (L.group_size == 32 || L.group_size == 64 || L.group_size == 128) &&
              L.group_size <= L.head_dim;
  bool p_ok = L.page_size % 64 == 0 && L.page_size <= 4096;
  return d_ok && g_ok && p_ok;
}
}  // namespace jfkv

// ------------------------------------------------------------------ pool
struct jf_page_pool {
  struct Seq {
    std::vector<int32_t> pages;
    int32_t length = 0;
    bool live = false;
  };
  int32_t num_pages = 0, page_size = 0;
  std::vector<int32_t> free_stack;  // may hold stale entries; in_free is the truth
  std::vector<uint8_t> in_free;
  std::vector<int32_t> refcount;
  int32_t n_free = 0, used = 0, high_water = 0;
  std::vector<Seq> seqs;

  int32_t pop_free() {
    while (!free_stack.empty()) {
      int32_t p = free_stack.back();
      free_stack.pop_back();
      if (in_free[p]) {
        in_free[p] = 0;
        --n_free;
        return p;
      }
    }
    return -1;
  }
  void push_free(int32_t p) {
    in_free[p] = 1;
    ++n_free;
    free_stack.push_back(p);
  }
  void take_ref(int32_t p) {
    if (refcount[p]++ == 0) {
      ++used;
      if (used > high_water) high_water = used;
    }
  }
  void drop_ref(int32_t p) {
    if (--refcount[p] == 0) {
      --used;
      push_free(p);
    }
  }
  Seq* get(int32_t s) {
    if (s < 0 || s >= (int32_t)seqs.size() || !seqs[s].live) return nullptr;
    return &seqs[s];
  }
  const Seq* get(int32_t s) const {
    if (s < 0 || s >= (int32_t)seqs.size() || !seqs[s].live) return nullptr;
    return &seqs[s];
  }
  int32_t new_seq() {
    seqs.emplace_back();
    seqs.back().live = true;
    return (int32_t)seqs.size() - 1;
  }
};

extern "C" {

const char* jf_last_error(void) { return g_last_error.c_str(); }

const char* jf_version(void) { return "jfkv 0.1 (gfx950)"; }

jf_status jf_kv_pool_bytes(const jf_kv_layout* layout, size_t* codes_bytes,
                           size_t* meta_bytes) {
  jf_status st = check_layout(layout);
  if (st) return st;
  if (!codes_bytes || !meta_bytes) return fail(JF_ERR_INVALID, "NULL output");
  size_t per = (size_t)layout->num_pages * layout->num_kv_heads * layout->page_size;
  *codes_bytes = per * (size_t)(layout->head_dim / 2);
  *meta_bytes = per * (size_t)(layout->head_dim / layout->group_size) * 2 * sizeof(uint16_t);
  return ok();
}

jf_status jf_page_table_pool_create(int32_t num_pages, int32_t page_size,
                                    uint64_t shuffle_seed, jf_page_pool** out) {
  if (!out) return fail(JF_ERR_INVALID, "out is NULL");
  if (num_pages <= 0 || page_size <= 0)
    return fail(JF_ERR_INVALID, "num_pages and page_size must be positive");
  jf_page_pool* p = new (std::nothrow) jf_page_pool;
  if (!p) return fail(JF_ERR_INVALID, "out of host memory");
  try {
    p->num_pages = num_pages;
    p->page_size = page_size;
    p->in_free.assign(num_pages, 1);
    p->refcount.assign(num_pages, 0);
    std::vector<int32_t> order(num_pages);
    for (int32_t i = 0; i < num_pages; ++i) order[i] = i;
    if (shuffle_seed) {
      uint64_t s = shuffle_seed;
      for (int32_t i = num_pages - 1; i > 0; --i) {  // Fisher-Yates
        int32_t j = (int32_t)(splitmix64(s) % (uint64_t)(i + 1));
        std::swap(order[i], order[j]);
      }
    }
    // the stack pops from the back: hand pages out in `order`
    p->free_stack.assign(order.rbegin(), order.rend());
    p->n_free = num_pages;
  } catch (...) {
    delete p;
    return fail(JF_ERR_INVALID, "out of host memory");
  }
  *out = p;
  return ok();
}

jf_status jf_page_table_pool_destroy(jf_page_pool* pool) {
  if (!pool) return fail(JF_ERR_INVALID, "pool is NULL");
  delete pool;
  return ok();
}

jf_status jf_page_table_create(jf_page_pool* pool, int32_t* seq) {
  if (!pool || !seq) return fail(JF_ERR_INVALID, "NULL argument");
  *seq = pool->new_seq();
  return ok();
}

jf_status jf_page_table_fork(jf_page_pool* pool, int32_t src, int32_t prefix_len,
                             int32_t* seq) {
  if (!pool || !seq) return fail(JF_ERR_INVALID, "NULL argument");
  const jf_page_pool::Seq* s = pool->get(src);
  if (!s) return fail(JF_ERR_STATE, "fork: unknown or released request %d", src);
  if (prefix_len < 0 || prefix_len % pool->page_size || prefix_len > s->length)
    return fail(JF_ERR_INVALID,
                "fork: prefix_len %d must be a multiple of page_size %d and <= length %d",
                prefix_len, pool->page_size, s->length);
  int32_t np = prefix_len / pool->page_size;
  std::vector<int32_t> pages(s->pages.begin(), s->pages.begin() + np);
  int32_t id = pool->new_seq();
  for (int32_t pg : pages) pool->take_ref(pg);
  pool->seqs[id].pages = std::move(pages);
  pool->seqs[id].length = prefix_len;
  *seq = id;
  return ok();
}

jf_status jf_page_table_assign(jf_page_pool* pool, int32_t seq, const int32_t* page_ids,
                               int32_t n) {
  if (!pool || (n > 0 && !page_ids) || n < 0) return fail(JF_ERR_INVALID, "bad argument");
  jf_page_pool::Seq* s = pool->get(seq);
  if (!s) return fail(JF_ERR_STATE, "assign: unknown or released request %d", seq);
  std::vector<uint8_t> seen(pool->num_pages, 0);
  for (int32_t i = 0; i < n; ++i) {
    int32_t p = page_ids[i];
    if (p < 0 || p >= pool->num_pages)
      return fail(JF_ERR_INVALID, "assign: page %d out of range", p);
    if (!pool->in_free[p] || seen[p])
      return fail(JF_ERR_STATE, "assign: page %d is not free", p);
    seen[p] = 1;
  }
  for (int32_t i = 0; i < n; ++i) {
    int32_t p = page_ids[i];
    pool->in_free[p] = 0;  // its stack entry goes stale
    --pool->n_free;
    pool->take_ref(p);
    s->pages.push_back(p);
  }
  return ok();
}

jf_status jf_page_table_reserve(jf_page_pool* pool, int32_t seq, int32_t new_len) {
  if (!pool) return fail(JF_ERR_INVALID, "pool is NULL");
  jf_page_pool::Seq* s = pool->get(seq);
  if (!s) return fail(JF_ERR_STATE, "reserve: unknown or released request %d", seq);
  if (new_len < 0) return fail(JF_ERR_INVALID, "reserve: negative length");
  const int32_t P = pool->page_size;
  int64_t need_pages = ((int64_t)new_len + P - 1) / P;
  if (new_len > s->length) {
    // positions length..new_len-1 that land on pages already held must not
    // be on shared pages
    int64_t first = s->length / P;
    int64_t last = std::min<int64_t>(need_pages, (int64_t)s->pages.size());
    for (int64_t lp = first; lp < last; ++lp)
      if (pool->refcount[s->pages[lp]] > 1)
        return fail(JF_ERR_STATE, "reserve: logical page %lld of request %d is shared",
                    (long long)lp, seq);
  }
  int64_t missing = need_pages - (int64_t)s->pages.size();
  if (missing <= 0) return ok();
  if (missing > pool->n_free)
    return fail(JF_ERR_NO_PAGES, "reserve: need %lld pages, %d free", (long long)missing,
                pool->n_free);
  for (int64_t i = 0; i < missing; ++i) {
    int32_t p = pool->pop_free();
    pool->take_ref(p);
    s->pages.push_back(p);
  }
  return ok();
}

jf_status jf_page_table_set_length(jf_page_pool* pool, int32_t seq, int32_t len) {
  if (!pool) return fail(JF_ERR_INVALID, "pool is NULL");
  jf_page_pool::Seq* s = pool->get(seq);
  if (!s) return fail(JF_ERR_STATE, "set_length: unknown or released request %d", seq);
  if (len < 0 || (int64_t)len > (int64_t)s->pages.size() * pool->page_size)
    return fail(JF_ERR_INVALID, "set_length: %d exceeds the capacity of %zu pages", len,
                s->pages.size());
  s->length = len;
  return ok();
}

jf_status jf_page_table_release(jf_page_pool* pool, int32_t seq) {
  if (!pool) return fail(JF_ERR_INVALID, "pool is NULL");
  jf_page_pool::Seq* s = pool->get(seq);
  if (!s) return fail(JF_ERR_STATE, "release: unknown or released request %d", seq);
  for (int32_t p : s->pages) pool->drop_ref(p);
  s->pages.clear();
  s->pages.shrink_to_fit();
  s->length = 0;
  s->live = false;
  return ok();
}

jf_status jf_page_table_export(const jf_page_pool* pool, const int32_t* seqs, int32_t n,
                               int32_t max_pages, int32_t* block_table, int32_t* lens) {
  if (!pool || (n > 0 && (!seqs || !block_table || !lens)) || n < 0 || max_pages < 0)
    return fail(JF_ERR_INVALID, "bad argument");
  for (int32_t i = 0; i < n; ++i) {
    const jf_page_pool::Seq* s = pool->get(seqs[i]);
    if (!s) return fail(JF_ERR_STATE, "export: unknown or released request %d", seqs[i]);
    if ((int64_t)s->pages.size() > max_pages)
      return fail(JF_ERR_INVALID, "export: request %d has %zu pages > max_pages %d", seqs[i],
                  s->pages.size(), max_pages);
  }
  for (int32_t i = 0; i < n; ++i) {
    const jf_page_pool::Seq* s = pool->get(seqs[i]);
    int32_t* row = block_table + (size_t)i * max_pages;
    size_t k = 0;
    for (; k < s->pages.size(); ++k) row[k] = s->pages[k];
    for (; k < (size_t)max_pages; ++k) row[k] = -1;
    lens[i] = s->length;
  }
  return ok();
}

jf_status jf_page_table_stats(const jf_page_pool* pool, int32_t* free_pages,
                              int32_t* used_pages, int32_t* high_water) {
  if (!pool || !free_pages || !used_pages || !high_water)
    return fail(JF_ERR_INVALID, "NULL argument");
  *free_pages = pool->n_free;
  *used_pages = pool->used;
  *high_water = pool->high_water;
  return ok();
}

jf_status jf_page_table_info(const jf_page_pool* pool, int32_t seq, int32_t* n_pages,
                             int32_t* length) {
  if (!pool || !n_pages || !length) return fail(JF_ERR_INVALID, "NULL argument");
  const jf_page_pool::Seq* s = pool->get(seq);
  if (!s) return fail(JF_ERR_STATE, "info: unknown or released request %d", seq);
  *n_pages = (int32_t)s->pages.size();
  *length = s->length;
  return ok();
}

// ------------------------------------------------------------------ device
jf_status jf_kv_quantize_append(const jf_kv_layout* layout, const jf_kv_pool_ptrs* pool,
                                const void* k_new, const void* v_new, const int32_t* cu_tok,
                                const int32_t* start_pos, const int32_t* block_tables,
                                int32_t B, int32_t max_pages, int32_t total_tok,
                                hipStream_t stream) {
  jf_status st = check_layout(layout);
  if (st) return st;
  if ((st = check_pool(pool))) return st;
  if (B <= 0 || max_pages <= 0 || total_tok < 0)
    return fail(JF_ERR_INVALID, "B and max_pages must be positive, total_tok >= 0");
  if (total_tok == 0) return ok();
  if (!k_new || !v_new || !cu_tok || !start_pos || !block_tables)
    return fail(JF_ERR_INVALID, "NULL device pointer");
  return device_status(jfkv::launch_quantize_append(*layout, *pool, k_new, v_new, cu_tok,
                                                    start_pos, block_tables, B, max_pages,
                                                    total_tok, stream),
                       "quantize_append launch");
}

jf_status jf_decode_workspace_bytes(int32_t B, int32_t num_q_heads, int32_t head_dim,
                                    int32_t max_splits, size_t* bytes) {
  if (!bytes || B <= 0 || num_q_heads <= 0 || head_dim <= 0 || max_splits <= 0 ||
      max_splits > 1024)
    return fail(JF_ERR_INVALID, "bad argument (max_splits must be 1..1024)");
  if ((int64_t)B * num_q_heads > jfkv::kDecodeMaxHeads)
    return fail(JF_ERR_UNSUPPORTED, "B * num_q_heads above %d", jfkv::kDecodeMaxHeads);
  *bytes = jfkv::decode_workspace_bytes(B, num_q_heads, head_dim, max_splits);
  return ok();
}

namespace {

// Arguments every decode entry point shares (everything but the workspace).
jf_status check_decode_args(const jf_kv_layout* layout, const jf_kv_pool_ptrs* pool,
                            const void* q, int32_t B, int32_t num_q_heads,
                            const int32_t* block_tables, int32_t max_pages,
                            const int32_t* seq_lens, float softmax_scale, int32_t max_splits,
                            void* out) {
  jf_status st = check_layout(layout);
  if (st) return st;
  if ((st = check_pool(pool))) return st;
  if (!q || !block_tables || !seq_lens || !out)
    return fail(JF_ERR_INVALID, "NULL device pointer");
  if (B <= 0 || num_q_heads <= 0 || max_pages <= 0)
    return fail(JF_ERR_INVALID, "B, num_q_heads and max_pages must be positive");
  if (num_q_heads % layout->num_kv_heads)
    return fail(JF_ERR_INVALID, "num_q_heads %d is not a multiple of num_kv_heads %d",
                num_q_heads, layout->num_kv_heads);
  if ((int64_t)max_pages * layout->page_size > INT32_MAX)
    return fail(JF_ERR_INVALID, "max_pages * page_size overflows int32");
  if (max_splits <= 0 || max_splits > 1024)
    return fail(JF_ERR_INVALID, "max_splits must be 1..1024");
  if (!(softmax_scale == softmax_scale) || softmax_scale == INFINITY ||
      softmax_scale == -INFINITY)
    return fail(JF_ERR_INVALID, "softmax_scale must be finite");
  return ok();
}

jf_status decode_common(const jf_kv_layout* layout, const jf_kv_pool_ptrs* pool,
                        const void* k_new, const void* v_new, const void* q, int32_t B,
                        int32_t num_q_heads, const int32_t* block_tables, int32_t max_pages,
                        const int32_t* seq_lens, float softmax_scale, int32_t max_splits,
                        void* workspace, size_t workspace_bytes, void* out, hipStream_t stream) {
  jf_status st = check_layout(layout);
  if (st) return st;
  if ((st = check_pool(pool))) return st;
  if (!q || !block_tables || !seq_lens || !workspace || !out)
    return fail(JF_ERR_INVALID, "NULL device pointer");
  if (B <= 0 || num_q_heads <= 0 || max_pages <= 0)
    return fail(JF_ERR_INVALID, "B, num_q_heads and max_pages must be positive");
  if (num_q_heads % layout->num_kv_heads)
    return fail(JF_ERR_INVALID, "num_q_heads %d is not a multiple of num_kv_heads %d",
                num_q_heads, layout->num_kv_heads);
  if ((int64_t)max_pages * layout->page_size > INT32_MAX)
    return fail(JF_ERR_INVALID, "max_pages * page_size overflows int32");
  size_t need = 0;
  if ((st = jf_decode_workspace_bytes(B, num_q_heads, layout->head_dim, max_splits, &need)))
    return st;
  if (workspace_bytes < need)
    return fail(JF_ERR_INVALID, "workspace %zu bytes < required %zu", workspace_bytes, need);
  if (!(softmax_scale == softmax_scale) || softmax_scale == INFINITY ||
      softmax_scale == -INFINITY)
    return fail(JF_ERR_INVALID, "softmax_scale must be finite");
  return device_status(jfkv::launch_decode(*layout, *pool, k_new, v_new, q, B, num_q_heads,
                                           block_tables, max_pages, seq_lens, softmax_scale,
                                           max_splits, workspace, out, stream),
                       "decode launch");
}

}  // namespace

jf_status jf_decode_attn_q4(const jf_kv_layout* layout, const jf_kv_pool_ptrs* pool,
                            const void* q, int32_t B, int32_t num_q_heads,
                            const int32_t* block_tables, int32_t max_pages,
                            const int32_t* seq_lens, float softmax_scale, int32_t max_splits,
                            void* workspace, size_t workspace_bytes, void* out,
                            hipStream_t stream) {
  return decode_common(layout, pool, nullptr, nullptr, q, B, num_q_heads, block_tables,
                       max_pages, seq_lens, softmax_scale, max_splits, workspace,
                       workspace_bytes, out, stream);
}

jf_status jf_verify_attn_q4(const jf_kv_layout* layout, const jf_kv_pool_ptrs* pool,
                            const void* q, int32_t B, int32_t num_queries, int32_t num_q_heads,
                            const int32_t* block_tables, int32_t max_pages,
                            const int32_t* seq_lens, float softmax_scale, int32_t max_splits,
                            void* workspace, size_t workspace_bytes, void* out,
                            hipStream_t stream) {
  jf_status st = check_decode_args(layout, pool, q, B, num_q_heads, block_tables, max_pages,
                                   seq_lens, softmax_scale, max_splits, out);
  if (st) return st;
  if (!workspace) return fail(JF_ERR_INVALID, "NULL device pointer");
  if (num_queries < 1 || num_queries > 4)
    return fail(JF_ERR_UNSUPPORTED, "num_queries %d outside 1..4", num_queries);
  const int64_t heads = (int64_t)num_q_heads * num_queries;
  if (heads > INT32_MAX) return fail(JF_ERR_INVALID, "num_q_heads * num_queries overflows");
  size_t need = 0;
  if ((st = jf_decode_workspace_bytes(B, (int32_t)heads, layout->head_dim, max_splits, &need)))
    return st;
  if (workspace_bytes < need)
    return fail(JF_ERR_INVALID, "workspace %zu bytes < required %zu", workspace_bytes, need);
  return device_status(jfkv::launch_decode(*layout, *pool, nullptr, nullptr, q, B, (int32_t)heads,
                                           block_tables, max_pages, seq_lens, softmax_scale,
                                           max_splits, workspace, out, stream, num_queries),
                       "verify launch");
}

jf_status jf_decode_step_q4(const jf_kv_layout* layout, const jf_kv_pool_ptrs* pool,
                            const void* k_new, const void* v_new, const void* q, int32_t B,
                            int32_t num_q_heads, const int32_t* block_tables,
                            int32_t max_pages, const int32_t* seq_lens, float softmax_scale,
                            int32_t max_splits, void* workspace, size_t workspace_bytes,
                            void* out, hipStream_t stream) {
  if (!k_new || !v_new) return fail(JF_ERR_INVALID, "NULL device pointer");
  return decode_common(layout, pool, k_new, v_new, q, B, num_q_heads, block_tables, max_pages,
                       seq_lens, softmax_scale, max_splits, workspace, workspace_bytes, out,
                       stream);
}

jf_status jf_decode_step_q4_static(const jf_kv_layout* layout, const jf_kv_pool_ptrs* pool,
                                   const void* k_new, const void* v_new, const void* q,
                                   int32_t B, int32_t num_q_heads, const int32_t* block_tables,
                                   int32_t max_pages, const int32_t* seq_lens,
                                   float softmax_scale, int32_t max_splits, void* out,
                                   hipStream_t stream) {
  if (!k_new || !v_new) return fail(JF_ERR_INVALID, "NULL device pointer");
  jf_status st = check_decode_args(layout, pool, q, B, num_q_heads, block_tables, max_pages,
                                   seq_lens, softmax_scale, max_splits, out);
  if (st) return st;
  const int64_t gq = num_q_heads / layout->num_kv_heads;
  const int64_t tickets = (int64_t)B * layout->num_kv_heads * ((gq + 3) / 4);
  const int64_t records = (int64_t)B * num_q_heads * max_splits * (layout->head_dim + 4) *
                          (int64_t)sizeof(float);
  const int64_t room = (int64_t)(jfkv::kStaticScratchBytes - jfkv::kStaticTicketBytes);
  if (tickets > jfkv::kStaticTickets || records > room)
    return fail(JF_ERR_INVALID,
                "jf_decode_step_q4_static: B = %d, num_q_heads = %d, max_splits = %d need %lld "
                "counters and %lld bytes of split records; the static scratch holds %lld "
                "counters and %lld bytes (use jf_decode_step_q4 with a workspace)",
                B, num_q_heads, max_splits, (long long)tickets, (long long)records,
                (long long)jfkv::kStaticTickets, (long long)room);
  return device_status(jfkv::launch_decode_static(*layout, *pool, k_new, v_new, q, B,
                                                  num_q_heads, block_tables, max_pages,
                                                  seq_lens, softmax_scale, max_splits, out,
                                                  stream),
                       "decode launch (static scratch)");
}

jf_status jf_prefill_attn_q4(const jf_kv_layout* layout, const jf_kv_pool_ptrs* pool,
                             const void* q, const void* k_chunk, const void* v_chunk,
                             int32_t T, int32_t num_q_heads, const int32_t* block_table,
                             int32_t max_pages, int32_t prefix_len, float softmax_scale,
                             void* out, hipStream_t stream) {
  jf_status st = check_layout(layout);
  if (st) return st;
  if ((st = check_pool(pool))) return st;
  if (T < 0 || prefix_len < 0 || num_q_heads <= 0 || max_pages < 0)
    return fail(JF_ERR_INVALID, "negative size");
  if (num_q_heads % layout->num_kv_heads)
    return fail(JF_ERR_INVALID, "num_q_heads %d is not a multiple of num_kv_heads %d",
                num_q_heads, layout->num_kv_heads);
  if ((int64_t)prefix_len > (int64_t)max_pages * layout->page_size)
    return fail(JF_ERR_INVALID, "prefix_len %d exceeds max_pages %d * page_size %d",
                prefix_len, max_pages, layout->page_size);
  if ((int64_t)prefix_len + T > INT32_MAX)
    return fail(JF_ERR_INVALID, "prefix_len + T overflows int32");
  if (!(softmax_scale == softmax_scale) || softmax_scale == INFINITY ||
      softmax_scale == -INFINITY)
    return fail(JF_ERR_INVALID, "softmax_scale must be finite");
  if (T == 0) return ok();
  if (!q || !k_chunk || !v_chunk || !out || (prefix_len > 0 && !block_table))
    return fail(JF_ERR_INVALID, "NULL device pointer");
  return device_status(jfkv::launch_prefill(*layout, *pool, q, k_chunk, v_chunk, T,
                                            num_q_heads, block_table, max_pages, prefix_len,
                                            softmax_scale, out, stream),
                       "prefill launch");
}

namespace {

// Arguments of the page -> operand reconstructions (both formats).
jf_status check_reconstruct_args(const jf_kv_layout* layout, const int32_t* block_table,
                                 int32_t max_pages, int32_t n_pos, int32_t kv0,
                                 int32_t num_heads, void* k_out, void* v_out, uintptr_t align) {
  if (max_pages <= 0 || n_pos < 0)
    return fail(JF_ERR_INVALID, "max_pages must be positive and n_pos >= 0");
  if ((int64_t)n_pos > (int64_t)max_pages * layout->page_size)
    return fail(JF_ERR_INVALID, "n_pos %d exceeds max_pages %d * page_size %d", n_pos, max_pages,
                layout->page_size);
  if (kv0 < 0 || num_heads <= 0 || (int64_t)kv0 + num_heads > layout->num_kv_heads)
    return fail(JF_ERR_INVALID, "KV heads %d .. %d outside 0 .. %d", kv0, kv0 + num_heads - 1,
                layout->num_kv_heads - 1);
  if ((int64_t)num_heads * n_pos > INT32_MAX)
    return fail(JF_ERR_UNSUPPORTED, "num_heads * n_pos above INT32_MAX vectors");
  if (n_pos > 0 && (!block_table || !k_out || !v_out))
    return fail(JF_ERR_INVALID, "NULL device pointer");
  if (((uintptr_t)k_out | (uintptr_t)v_out) & (align - 1))
    return fail(JF_ERR_INVALID, "k_out and v_out must be %d-byte aligned", (int)align);
  return ok();
}

}  // namespace

jf_status jf_reconstruct_q4(const jf_kv_layout* layout, const jf_kv_pool_ptrs* pool,
                            const int32_t* block_table, int32_t max_pages, int32_t n_pos,
                            int32_t kv0, int32_t num_heads, void* k_out, void* v_out,
                            hipStream_t stream) {
  jf_status st = check_layout(layout);
  if (st) return st;
  if ((st = check_pool(pool))) return st;
  if ((st = check_reconstruct_args(layout, block_table, max_pages, n_pos, kv0, num_heads, k_out,
                                   v_out, 16)))
    return st;
  if ((((uintptr_t)pool->k_codes | (uintptr_t)pool->v_codes) & 15) ||
      (((uintptr_t)pool->k_meta | (uintptr_t)pool->v_meta) & 3))
    return fail(JF_ERR_INVALID, "pool codes must be 16-byte and meta 4-byte aligned");
  if (n_pos == 0) return ok();
  return device_status(jfkv::launch_reconstruct(*layout, *pool, block_table, max_pages, n_pos,
                                                kv0, num_heads, k_out, v_out, stream),
                       "reconstruct launch");
}

// ------------------------------------------------------------------ TQ4
namespace {

jf_status check_tq4_layout(const jf_kv_layout* layout) {
  if (!layout) return fail(JF_ERR_INVALID, "layout is NULL");
  if (layout->page_size <= 0 || layout->num_kv_heads <= 0 || layout->num_pages <= 0)
    return fail(JF_ERR_INVALID, "page_size, num_kv_heads and num_pages must be positive");
  if (layout->head_dim != 256)
    return fail(JF_ERR_UNSUPPORTED, "TQ4 head_dim must be 256, got %d", layout->head_dim);
  if ((int64_t)layout->num_pages * layout->num_kv_heads * layout->page_size > INT32_MAX)
    return fail(JF_ERR_INVALID, "pool has more than INT32_MAX vectors");
  return ok();
}

}  // namespace

jf_status jf_tq4_pool_bytes(const jf_kv_layout* layout, size_t* words_bytes,
                            size_t* norms_bytes) {
  jf_status st = check_tq4_layout(layout);
  if (st) return st;
  if (!words_bytes || !norms_bytes) return fail(JF_ERR_INVALID, "NULL output pointer");
  const size_t vecs = (size_t)layout->num_pages * layout->num_kv_heads * layout->page_size;
  *words_bytes = vecs * (layout->head_dim / 2);
  *norms_bytes = vecs * 2;
  return ok();
}

jf_status jf_tq4_encode_append(const jf_kv_layout* layout, void* words, void* norms,
                               const void* x, const float* signs, const float* centroids,
                               const int32_t* cu_tok, const int32_t* start_pos,
                               const int32_t* block_tables, int32_t B, int32_t max_pages,
                               int32_t total_tok, hipStream_t stream) {
  jf_status st = check_tq4_layout(layout);
  if (st) return st;
  if (B <= 0 || max_pages <= 0 || total_tok < 0)
    return fail(JF_ERR_INVALID, "B and max_pages must be positive, total_tok >= 0");
  if (!words || !norms) return fail(JF_ERR_INVALID, "NULL pool pointer");
  if (total_tok == 0) return ok();
  if ((int64_t)total_tok * layout->num_kv_heads > INT32_MAX)
    return fail(JF_ERR_UNSUPPORTED, "total_tok * num_kv_heads above INT32_MAX vectors");
  if ((int64_t)max_pages * layout->page_size > INT32_MAX)
    return fail(JF_ERR_INVALID, "max_pages * page_size overflows int32");
  if (!x || !signs || !centroids || !cu_tok || !start_pos || !block_tables)
    return fail(JF_ERR_INVALID, "NULL device pointer");
  if (((uintptr_t)x & 7) || ((uintptr_t)signs & 15) || ((uintptr_t)words & 3) ||
      ((uintptr_t)norms & 1))
    return fail(JF_ERR_INVALID, "x must be 8-byte, signs 16-byte, words 4-byte, norms 2-byte aligned");
  return device_status(jfkv::launch_tq4_encode(*layout, words, norms, x, signs, centroids, cu_tok,
                                               start_pos, block_tables, B, max_pages, total_tok,
                                               stream),
                       "tq4_encode launch");
}

jf_status jf_tq4_decode_attn(const jf_kv_layout* layout, const void* k_words,
                             const void* k_norms, const void* v_words, const void* v_norms,
                             const float* k_signs, const float* v_signs, const float* centroids,
                             const void* q, int32_t B, int32_t num_q_heads,
                             const int32_t* block_tables, int32_t max_pages,
                             const int32_t* seq_lens, float softmax_scale, int32_t max_splits,
                             void* workspace, size_t workspace_bytes, void* out,
                             hipStream_t stream) {
  jf_status st = check_tq4_layout(layout);
  if (st) return st;
  if (layout->page_size % 32)
    return fail(JF_ERR_UNSUPPORTED, "TQ4 decode needs page_size a multiple of 32, got %d",
                layout->page_size);
  if (!k_words || !k_norms || !v_words || !v_norms || !k_signs || !v_signs || !centroids || !q ||
      !block_tables || !seq_lens || !workspace || !out)
    return fail(JF_ERR_INVALID, "NULL device pointer");
  if (B <= 0 || num_q_heads <= 0 || max_pages <= 0)
    return fail(JF_ERR_INVALID, "B, num_q_heads and max_pages must be positive");
  if (num_q_heads % layout->num_kv_heads)
    return fail(JF_ERR_INVALID, "num_q_heads %d is not a multiple of num_kv_heads %d",
                num_q_heads, layout->num_kv_heads);
  if (num_q_heads / layout->num_kv_heads > 16)
    return fail(JF_ERR_UNSUPPORTED, "TQ4 decode takes at most 16 query heads per KV head");
  if ((int64_t)max_pages * layout->page_size > INT32_MAX)
    return fail(JF_ERR_INVALID, "max_pages * page_size overflows int32");
  if (((uintptr_t)k_words | (uintptr_t)v_words | (uintptr_t)k_norms | (uintptr_t)v_norms) & 15)
    return fail(JF_ERR_INVALID, "index words and norms must be 16-byte aligned");
  size_t need = 0;
  if ((st = jf_decode_workspace_bytes(B, num_q_heads, layout->head_dim, max_splits, &need)))
    return st;
  if (workspace_bytes < need)
    return fail(JF_ERR_INVALID, "workspace %zu bytes < required %zu", workspace_bytes, need);
  if (!(softmax_scale == softmax_scale) || softmax_scale == INFINITY ||
      softmax_scale == -INFINITY)
    return fail(JF_ERR_INVALID, "softmax_scale must be finite");
  return device_status(jfkv::launch_tq4_decode(*layout, k_words, k_norms, v_words, v_norms,
                                               k_signs, v_signs, centroids, q, B, num_q_heads,
                                               block_tables, max_pages, seq_lens, softmax_scale,
                                               max_splits, workspace, out, stream),
                       "tq4_decode launch");
}

jf_status jf_tq4_reconstruct(const jf_kv_layout* layout, const void* k_words,
                             const void* k_norms, const void* v_words, const void* v_norms,
                             const float* k_signs, const float* v_signs, const float* centroids,
                             const int32_t* block_table, int32_t max_pages, int32_t n_pos,
                             int32_t kv0, int32_t num_heads, void* k_out, void* v_out,
                             hipStream_t stream) {
  jf_status st = check_tq4_layout(layout);
  if (st) return st;
  if ((st = check_reconstruct_args(layout, block_table, max_pages, n_pos, kv0, num_heads, k_out,
                                   v_out, 8)))
    return st;
  if (n_pos == 0) return ok();
  if (!k_words || !k_norms || !v_words || !v_norms || !k_signs || !v_signs || !centroids)
    return fail(JF_ERR_INVALID, "NULL device pointer");
  if ((((uintptr_t)k_words | (uintptr_t)v_words) & 3) ||
      (((uintptr_t)k_norms | (uintptr_t)v_norms) & 1) ||
      (((uintptr_t)k_signs | (uintptr_t)v_signs) & 15))
    return fail(JF_ERR_INVALID, "index words 4-byte, norms 2-byte, signs 16-byte aligned");
  return device_status(jfkv::launch_tq4_reconstruct(*layout, k_words, k_norms, v_words, v_norms,
                                                    k_signs, v_signs, centroids, block_table,
                                                    n_pos, kv0, num_heads, k_out, v_out, stream),
                       "tq4_reconstruct launch");
}

// ------------------------------------------------------------------ snapshots
namespace {

jf_status check_pool_aligned(const jf_kv_pool_ptrs* p) {
  jf_status st = check_pool(p);
  if (st) return st;
  if ((((uintptr_t)p->k_codes | (uintptr_t)p->v_codes) & 15) ||
      (((uintptr_t)p->k_meta | (uintptr_t)p->v_meta) & 3))
    return fail(JF_ERR_INVALID, "pool codes must be 16-byte and meta 4-byte aligned");
  return ok();
}

// Whether p is device memory (false also when the runtime cannot tell).
// Kernels never dereference host memory: a host allocation is usable on the
// device only through the device pointer of a mapped allocation.
bool is_device_memory(const void* p) {
  hipPointerAttribute_t a;
  if (hipPointerGetAttributes(&a, p) != hipSuccess) {
    (void)hipGetLastError();
    return false;
  }
  return a.type == hipMemoryTypeDevice;
}

bool is_pinned_host_memory(const void* p) {
  hipPointerAttribute_t a;
  if (hipPointerGetAttributes(&a, p) != hipSuccess) {
    (void)hipGetLastError();
    return false;
  }
  return a.type == hipMemoryTypeHost;
}

jf_status page_copy(const jf_kv_layout* layout, const jf_kv_pool_ptrs* pool,
                    const int32_t* block_table, int32_t first, int32_t count, const void* buf,
                    bool unpack, hipStream_t stream) {
  jf_status st = check_layout(layout);
  if (st) return st;
  if ((st = check_pool_aligned(pool))) return st;
  if (first < 0 || count < 0 || (int64_t)first + count > INT32_MAX)
    return fail(JF_ERR_INVALID, "first and count must be >= 0");
  if (count == 0) return ok();
  if (!block_table || !buf) return fail(JF_ERR_INVALID, "NULL pointer");
  if ((uintptr_t)buf & 15) return fail(JF_ERR_INVALID, "buf must be 16-byte aligned");
  if (!is_device_memory(buf)) return fail(JF_ERR_INVALID, "buf must be device memory");
  return device_status(jfkv::launch_page_runs(*layout, *pool, block_table, first, count,
                                              const_cast<void*>(buf), unpack, stream),
                       unpack ? "unpack_pages launch" : "pack_pages launch");
}

// The safetensors header of a snapshot: one U8 tensor per layer holding its
// pages in logical order; the layout and length as metadata (strings, as
// the format requires); padded with spaces to a multiple of 8 bytes.
std::string snapshot_header(const jf_kv_layout& L, int32_t n_layers, int32_t n_pos, size_t pb) {
  const int64_t n_pages = ((int64_t)n_pos + L.page_size - 1) / L.page_size;
  char buf[512];
  snprintf(buf, sizeof(buf),
           "{\"__metadata__\":{\"format\":\"jfkv-pages-1\",\"page_size\":\"%d\","
           "\"num_kv_heads\":\"%d\",\"head_dim\":\"%d\",\"group_size\":\"%d\","
           "\"n_layers\":\"%d\",\"n_pos\":\"%d\",\"page_bytes\":\"%zu\"}",
           L.page_size, L.num_kv_heads, L.head_dim, L.group_size, n_layers, n_pos, pb);
  std::string h = buf;
  const uint64_t layer_bytes = (uint64_t)n_pages * pb;
  for (int32_t l = 0; l < n_layers; ++l) {
    snprintf(buf, sizeof(buf),
             ",\"layer%d\":{\"dtype\":\"U8\",\"shape\":[%lld,%zu],\"data_offsets\":[%llu,%llu]}",
             l, (long long)n_pages, pb, (unsigned long long)(l * layer_bytes),
             (unsigned long long)((l + 1) * layer_bytes));
    h += buf;
  }
  h += "}";
  while (h.size() % 8) h += ' ';
  return h;
}

bool write_all(int fd, const void* p, size_t n) {
  const char* c = static_cast<const char*>(p);
  while (n > 0) {
    const ssize_t w = ::write(fd, c, n);
    if (w < 0) {
      if (errno == EINTR) continue;
      return false;
    }
    c += w;
    n -= (size_t)w;
  }
  return true;
}

bool pread_all(int fd, void* p, size_t n, off_t off) {
  char* c = static_cast<char*>(p);
  while (n > 0) {
    const ssize_t r = ::pread(fd, c, n, off);
    if (r < 0) {
      if (errno == EINTR) continue;
      return false;
    }
    if (r == 0) return false;  // end of file
    c += r;
    n -= (size_t)r;
    off += r;
  }
  return true;
}

// Arguments shared by save and restore; pages_out = pages of n_pos.
jf_status check_snapshot_args(const char* path, const jf_kv_layout* layout,
                              const jf_kv_pool_ptrs* pools, int32_t n_layers,
                              const int32_t* block_table, const int32_t* block_table_host,
                              int32_t max_pages, void* staging_dev, void* staging,
                              size_t staging_bytes) {
  jf_status st = check_layout(layout);
  if (st) return st;
  if (!path || !pools || !staging || !staging_dev) return fail(JF_ERR_INVALID, "NULL pointer");
  if (n_layers <= 0) return fail(JF_ERR_INVALID, "n_layers must be positive");
  for (int32_t l = 0; l < n_layers; ++l)
    if ((st = check_pool_aligned(&pools[l]))) return st;
  if (max_pages < 0) return fail(JF_ERR_INVALID, "max_pages must be >= 0");
  if (max_pages > 0 && (!block_table || !block_table_host))
    return fail(JF_ERR_INVALID, "NULL block table");
  if (((uintptr_t)staging | (uintptr_t)staging_dev) & 15)
    return fail(JF_ERR_INVALID, "staging buffers must be 16-byte aligned");
  const size_t pb = jfkv::page_bytes(*layout);
  if (staging_bytes / 2 < pb)
    return fail(JF_ERR_INVALID, "staging of %zu bytes holds less than two pages of %zu bytes",
                staging_bytes, pb);
  return ok();
}

// The staging buffers' kinds (asked of the runtime, after every other check).
jf_status check_staging_kinds(const void* staging_dev, const void* staging) {
  if (!is_device_memory(staging_dev))
    return fail(JF_ERR_INVALID, "staging_dev must be device memory");
  if (!is_pinned_host_memory(staging))
    return fail(JF_ERR_INVALID, "staging must be pinned host memory");
  return ok();
}

// Two events that alternate with the staging halves.
struct EventPair {
  hipEvent_t e[2] = {nullptr, nullptr};
  hipError_t create() {
    for (auto& x : e) {
      hipError_t r = hipEventCreateWithFlags(&x, hipEventDisableTiming);
      if (r != hipSuccess) return r;
    }
    return hipSuccess;
  }
  ~EventPair() {
    for (auto& x : e)
      if (x) (void)hipEventDestroy(x);
  }
};

}  // namespace

jf_status jf_kv_page_bytes(const jf_kv_layout* layout, size_t* bytes) {
  jf_status st = check_layout(layout);
  if (st) return st;
  if (!bytes) return fail(JF_ERR_INVALID, "NULL output pointer");
  *bytes = jfkv::page_bytes(*layout);
  return ok();
}

jf_status jf_calib_read_stream(const void* buf, size_t bytes, int32_t blocks, void* sink,
                               hipStream_t stream) {
  if (!buf || !sink) return fail(JF_ERR_INVALID, "NULL pointer");
  if (bytes == 0 || bytes % 16) return fail(JF_ERR_INVALID, "bytes must be a positive multiple of 16");
  if ((uintptr_t)buf & 15) return fail(JF_ERR_INVALID, "buf must be 16-byte aligned");
  if ((uintptr_t)sink & 3) return fail(JF_ERR_INVALID, "sink must be 4-byte aligned");
  if (blocks < 1 || blocks > 65535) return fail(JF_ERR_INVALID, "blocks must be 1 .. 65535");
  if (!is_device_memory(buf) || !is_device_memory(sink))
    return fail(JF_ERR_INVALID, "buf and sink must be device memory");
  return device_status(jfkv::launch_read_stream(buf, bytes, blocks, static_cast<uint32_t*>(sink),
                                                stream),
                       "read_stream launch");
}

jf_status jf_kv_pack_pages(const jf_kv_layout* layout, const jf_kv_pool_ptrs* pool,
                           const int32_t* block_table, int32_t first, int32_t count, void* buf,
                           hipStream_t stream) {
  return page_copy(layout, pool, block_table, first, count, buf, false, stream);
}

jf_status jf_kv_unpack_pages(const jf_kv_layout* layout, const jf_kv_pool_ptrs* pool,
                             const int32_t* block_table, int32_t first, int32_t count,
                             const void* buf, hipStream_t stream) {
  return page_copy(layout, pool, block_table, first, count, buf, true, stream);
}

jf_status jf_snapshot_save(const char* path, const jf_kv_layout* layout,
                           const jf_kv_pool_ptrs* pools, int32_t n_layers,
                           const int32_t* block_table, const int32_t* block_table_host,
                           int32_t max_pages, int32_t n_pos, void* staging_dev, void* staging,
                           size_t staging_bytes, hipStream_t stream) {
  jf_status st = check_snapshot_args(path, layout, pools, n_layers, block_table,
                                     block_table_host, max_pages, staging_dev, staging,
                                     staging_bytes);
  if (st) return st;
  const int32_t P = layout->page_size;
  if (n_pos < 0 || (int64_t)n_pos > (int64_t)max_pages * P)
    return fail(JF_ERR_INVALID, "n_pos %d outside 0 .. max_pages * page_size", n_pos);
  const int32_t n_pages = (int32_t)(((int64_t)n_pos + P - 1) / P);
  for (int32_t i = 0; i < n_pages; ++i)
    if (block_table_host[i] < 0 || block_table_host[i] >= layout->num_pages)
      return fail(JF_ERR_INVALID, "page %d of the request (ID %d) is not in the pool", i,
                  block_table_host[i]);
  if ((st = check_staging_kinds(staging_dev, staging))) return st;
  const size_t pb = jfkv::page_bytes(*layout);
  const int32_t per = (int32_t)std::min<size_t>(staging_bytes / 2 / pb, (size_t)INT32_MAX);
  const std::string header = snapshot_header(*layout, n_layers, n_pos, pb);
  const std::string tmp = std::string(path) + ".tmp";
  EventPair ev;
  if (hipError_t e = ev.create(); e != hipSuccess) return device_status(e, "hipEventCreate");
  const int fd = ::open(tmp.c_str(), O_WRONLY | O_CREAT | O_TRUNC | O_CLOEXEC, 0644);
  if (fd < 0) return fail(JF_ERR_IO, "open %s: %s", tmp.c_str(), strerror(errno));
  // on failure: let enqueued copies finish (the caller may free the staging
  // buffers), drop the temporary file
  auto abort_with = [&](jf_status s) {
    (void)hipStreamSynchronize(stream);
    ::close(fd);
    ::unlink(tmp.c_str());
    return s;
  };
  const uint64_t hl = header.size();
  uint8_t len8[8];
  for (int i = 0; i < 8; ++i) len8[i] = (uint8_t)(hl >> (8 * i));
  if (!write_all(fd, len8, 8) || !write_all(fd, header.data(), header.size()))
    return abort_with(fail(JF_ERR_IO, "write %s: %s", tmp.c_str(), strerror(errno)));
  // chunk c: pages packed into device half c % 2 by a kernel, copied to host
  // half c % 2 (stream order keeps a device half from being refilled before
  // its copy), written to the file while chunk c + 1 packs and copies
  uint8_t* dh[2] = {static_cast<uint8_t*>(staging_dev),
                    static_cast<uint8_t*>(staging_dev) + per * pb};
  uint8_t* hh[2] = {static_cast<uint8_t*>(staging), static_cast<uint8_t*>(staging) + per * pb};
  size_t pending = 0;  // bytes of the chunk copied last, not yet written
  int c = 0;
  for (int32_t l = 0; l < n_layers; ++l) {
    for (int32_t p0 = 0; p0 < n_pages; p0 += per, ++c) {
      const int32_t cnt = std::min(per, n_pages - p0);
      const int h = c & 1;
      const size_t nbytes = (size_t)cnt * pb;
      hipError_t e = jfkv::launch_page_runs(*layout, pools[l], block_table, p0, cnt, dh[h],
                                            false, stream);
      if (e == hipSuccess) e = hipMemcpyAsync(hh[h], dh[h], nbytes, hipMemcpyDeviceToHost, stream);
      if (e == hipSuccess) e = hipEventRecord(ev.e[h], stream);
      if (e != hipSuccess) return abort_with(device_status(e, "snapshot pack"));
      if (c > 0) {  // the previous chunk, in the other half
        if ((e = hipEventSynchronize(ev.e[h ^ 1])) != hipSuccess)
          return abort_with(device_status(e, "snapshot pack"));
        if (!write_all(fd, hh[h ^ 1], pending))
          return abort_with(fail(JF_ERR_IO, "write %s: %s", tmp.c_str(), strerror(errno)));
      }
      pending = nbytes;
    }
  }
  if (c > 0) {
    const int h = (c - 1) & 1;
    if (hipError_t e = hipEventSynchronize(ev.e[h]); e != hipSuccess)
      return abort_with(device_status(e, "snapshot pack"));
    if (!write_all(fd, hh[h], pending))
      return abort_with(fail(JF_ERR_IO, "write %s: %s", tmp.c_str(), strerror(errno)));
  }
  if (::fsync(fd) != 0)
    return abort_with(fail(JF_ERR_IO, "fsync %s: %s", tmp.c_str(), strerror(errno)));
  if (::close(fd) != 0) {
    ::unlink(tmp.c_str());
    return fail(JF_ERR_IO, "close %s: %s", tmp.c_str(), strerror(errno));
  }
  if (::rename(tmp.c_str(), path) != 0) {
    const int err = errno;
    ::unlink(tmp.c_str());
    return fail(JF_ERR_IO, "rename %s -> %s: %s", tmp.c_str(), path, strerror(err));
  }
  return ok();
}

jf_status jf_snapshot_restore(const char* path, const jf_kv_layout* layout,
                              const jf_kv_pool_ptrs* pools, int32_t n_layers,
                              const int32_t* block_table, const int32_t* block_table_host,
                              int32_t max_pages, void* staging_dev, void* staging,
                              size_t staging_bytes, int32_t* n_pos_out, hipStream_t stream) {
  jf_status st = check_snapshot_args(path, layout, pools, n_layers, block_table,
                                     block_table_host, max_pages, staging_dev, staging,
                                     staging_bytes);
  if (st) return st;
  if (!n_pos_out) return fail(JF_ERR_INVALID, "NULL output pointer");
  const int fd = ::open(path, O_RDONLY | O_CLOEXEC);
  if (fd < 0) return fail(JF_ERR_IO, "open %s: %s", path, strerror(errno));
  bool enqueued = false;
  auto done = [&](jf_status s) {
    if (enqueued) (void)hipStreamSynchronize(stream);
    ::close(fd);
    return s;
  };
  uint8_t len8[8];
  if (!pread_all(fd, len8, 8, 0)) return done(fail(JF_ERR_INVALID, "%s: no header", path));
  uint64_t hl = 0;
  for (int i = 0; i < 8; ++i) hl |= (uint64_t)len8[i] << (8 * i);
  if (hl == 0 || hl > (1u << 24)) return done(fail(JF_ERR_INVALID, "%s: bad header size", path));
  std::string header(hl, '\0');
  if (!pread_all(fd, &header[0], hl, 8)) return done(fail(JF_ERR_INVALID, "%s: short header", path));
  // the position count, then the whole header must be the one save writes
  const char* key = "\"n_pos\":\"";
  const size_t at = header.find(key);
  if (at == std::string::npos) return done(fail(JF_ERR_INVALID, "%s: not a snapshot", path));
  const long long np_ll = strtoll(header.c_str() + at + strlen(key), nullptr, 10);
  if (np_ll < 0 || np_ll > INT32_MAX) return done(fail(JF_ERR_INVALID, "%s: bad n_pos", path));
  const int32_t n_pos = (int32_t)np_ll;
  const size_t pb = jfkv::page_bytes(*layout);
  if (header != snapshot_header(*layout, n_layers, n_pos, pb))
    return done(fail(JF_ERR_INVALID,
                     "%s: not a snapshot of this layout and layer count (header differs)", path));
  const int32_t P = layout->page_size;
  const int32_t n_pages = (int32_t)(((int64_t)n_pos + P - 1) / P);
  struct stat sb;
  if (::fstat(fd, &sb) != 0) return done(fail(JF_ERR_IO, "stat %s: %s", path, strerror(errno)));
  const uint64_t data0 = 8 + hl;
  if ((uint64_t)sb.st_size != data0 + (uint64_t)n_layers * n_pages * pb)
    return done(fail(JF_ERR_INVALID, "%s: size %lld, expected %llu", path, (long long)sb.st_size,
                     (unsigned long long)(data0 + (uint64_t)n_layers * n_pages * pb)));
  if (n_pages > max_pages)
    return done(fail(JF_ERR_INVALID, "the snapshot has %d pages, the table %d", n_pages,
                     max_pages));
  {
    std::vector<int32_t> ids(block_table_host, block_table_host + n_pages);
    for (int32_t id : ids)
      if (id < 0 || id >= layout->num_pages)
        return done(fail(JF_ERR_INVALID, "page ID %d is not in the pool", id));
    std::sort(ids.begin(), ids.end());
    if (std::adjacent_find(ids.begin(), ids.end()) != ids.end())
      return done(fail(JF_ERR_INVALID, "the table lists a page twice"));
  }
  if ((st = check_staging_kinds(staging_dev, staging))) return done(st);
  EventPair ev;
  if (hipError_t e = ev.create(); e != hipSuccess) return done(device_status(e, "hipEventCreate"));
  const int32_t per = (int32_t)std::min<size_t>(staging_bytes / 2 / pb, (size_t)INT32_MAX);
  uint8_t* dh[2] = {static_cast<uint8_t*>(staging_dev),
                    static_cast<uint8_t*>(staging_dev) + per * pb};
  uint8_t* hh[2] = {static_cast<uint8_t*>(staging), static_cast<uint8_t*>(staging) + per * pb};
  // chunk c: read into host half c % 2 once its previous copy (chunk c - 2)
  // has left it, copied to device half c % 2, unpacked into the pages
  int c = 0;
  for (int32_t l = 0; l < n_layers; ++l) {
    for (int32_t p0 = 0; p0 < n_pages; p0 += per, ++c) {
      const int32_t cnt = std::min(per, n_pages - p0);
      const int h = c & 1;
      const size_t nbytes = (size_t)cnt * pb;
      hipError_t e = hipSuccess;
      if (c >= 2 && (e = hipEventSynchronize(ev.e[h])) != hipSuccess)
        return done(device_status(e, "snapshot unpack"));
      const off_t off = (off_t)(data0 + ((uint64_t)l * n_pages + p0) * pb);
      errno = 0;
      if (!pread_all(fd, hh[h], nbytes, off))
        return done(fail(JF_ERR_IO, "read %s: %s", path, errno ? strerror(errno) : "short"));
      enqueued = true;
      e = hipMemcpyAsync(dh[h], hh[h], nbytes, hipMemcpyHostToDevice, stream);
      if (e == hipSuccess) e = hipEventRecord(ev.e[h], stream);  // host half h free again
      if (e == hipSuccess)
        e = jfkv::launch_page_runs(*layout, pools[l], block_table, p0, cnt, dh[h], true, stream);
      if (e != hipSuccess) return done(device_status(e, "snapshot unpack"));
    }
  }
  if (hipError_t e = hipStreamSynchronize(stream); e != hipSuccess)
    return done(device_status(e, "snapshot unpack"));
  *n_pos_out = n_pos;
  ::close(fd);
  return ok();
}

}  // extern "C"
