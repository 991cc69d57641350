// Exercises the host side of libjfkv.so (page allocator, argument
// validation, the snapshot writer and reader) built with AddressSanitizer and
// UndefinedBehaviorSanitizer against the CPU stand-ins of stubs.cpp.  Exits
// non-zero on the first failed check; the sanitizers abort on their own
// findings.  Test infrastructure only.
#include <unistd.h>

#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <random>
#include <set>
#include <string>
#include <vector>

#include "jfkv.h"

void stub_register(const void* p, size_t n, bool device);
void stub_clear();

static int g_checks = 0;
#define CHECK(c)                                                                       \
  do {                                                                                 \
    ++g_checks;                                                                        \
    if (!(c)) {                                                                        \
      std::fprintf(stderr, "%s:%d: check failed: %s (last error: %s)\n", __FILE__,     \
                   __LINE__, #c, jf_last_error());                                     \
      std::exit(1);                                                                    \
    }                                                                                  \
  } while (0)

// Random operations on the page allocator; its accounting must stay
// consistent and every exported table must list distinct pages of the pool
// (shared prefixes aside).
static void page_table_fuzz() {
  const int32_t NP = 96, P = 64;
  jf_page_pool* pool = nullptr;
  CHECK(jf_page_table_pool_create(NP, P, 7, &pool) == JF_OK);
  std::mt19937 rng(1);
  std::vector<int32_t> live;
  std::vector<int32_t> lens;
  for (int op = 0; op < 4000; ++op) {
    const int k = rng() % 6;
    if (k == 0 || live.empty()) {
      int32_t s = -1;
      CHECK(jf_page_table_create(pool, &s) == JF_OK);
      live.push_back(s);
      lens.push_back(0);
    } else {
      const size_t i = rng() % live.size();
      const int32_t s = live[i];
      if (k == 1) {
        const int32_t want = lens[i] + (int32_t)(rng() % 300);
        const jf_status st = jf_page_table_reserve(pool, s, want);
        CHECK(st == JF_OK || st == JF_ERR_NO_PAGES);
        if (st == JF_OK) {
          CHECK(jf_page_table_set_length(pool, s, want) == JF_OK);
          lens[i] = want;
        }
      } else if (k == 2 && lens[i] >= P) {
        int32_t f = -1;
        const int32_t pre = P * (int32_t)(rng() % (lens[i] / P + 1));
        CHECK(jf_page_table_fork(pool, s, pre, &f) == JF_OK);
        live.push_back(f);
        lens.push_back(pre);
      } else if (k == 3) {
        CHECK(jf_page_table_release(pool, s) == JF_OK);
        live.erase(live.begin() + i);
        lens.erase(lens.begin() + i);
        int32_t np_ = 0, len_ = 0;
        CHECK(jf_page_table_info(pool, s, &np_, &len_) != JF_OK);  // released handle
      } else if (k == 4) {
        int32_t fp = 0, up = 0, hw = 0;
        CHECK(jf_page_table_stats(pool, &fp, &up, &hw) == JF_OK);
        CHECK(fp + up == NP && up <= hw && hw <= NP);
      } else {
        const int32_t n = (int32_t)live.size();
        const int32_t maxp = (int32_t)((4000 * 300) / P + 2);
        std::vector<int32_t> tab((size_t)n * 64, -2), ls(n);
        const jf_status st = jf_page_table_export(pool, live.data(), n, 64, tab.data(), ls.data());
        CHECK(st == JF_OK || st == JF_ERR_INVALID);
        (void)maxp;
        if (st == JF_OK)
          for (int32_t r = 0; r < n; ++r) {
            CHECK(ls[r] == lens[r]);
            for (int32_t j = 0; j < 64; ++j) CHECK(tab[(size_t)r * 64 + j] >= -1 && tab[(size_t)r * 64 + j] < NP);
          }
      }
    }
  }
  // bad handles and arguments
  int32_t s = -1;
  CHECK(jf_page_table_create(nullptr, &s) == JF_ERR_INVALID);
  CHECK(jf_page_table_reserve(pool, 123456, 10) != JF_OK);
  CHECK(jf_page_table_fork(pool, live.empty() ? 0 : live[0], 1, &s) != JF_OK);  // not page-aligned
  for (int32_t h : live) CHECK(jf_page_table_release(pool, h) == JF_OK);
  int32_t fp = 0, up = 0, hw = 0;
  CHECK(jf_page_table_stats(pool, &fp, &up, &hw) == JF_OK && fp == NP && up == 0);
  CHECK(jf_page_table_pool_destroy(pool) == JF_OK);
  CHECK(jf_page_table_pool_create(0, 64, 0, &pool) == JF_ERR_INVALID);
}

// Every device entry point rejects bad arguments before any launch, and
// accepts good ones (the stand-in launches do nothing).
static void validation() {
  jf_kv_layout L = {256, 8, 128, 64, 16};
  std::vector<uint8_t> mem(1 << 20);
  void* p = mem.data();
  jf_kv_pool_ptrs pool = {p, p, p, p};
  size_t ws = 0;
  CHECK(jf_decode_workspace_bytes(1, 32, 128, 8, &ws) == JF_OK);
  const int32_t* ip = reinterpret_cast<const int32_t*>(p);
  CHECK(jf_decode_attn_q4(&L, &pool, p, 1, 30, ip, 4, ip, 1.0f, 8, p, ws, p, nullptr) == JF_ERR_INVALID);
  CHECK(std::strstr(jf_last_error(), "multiple") != nullptr);
  CHECK(jf_decode_attn_q4(&L, &pool, p, 1, 32, ip, 4, ip, 1.0f, 8, p, 16, p, nullptr) == JF_ERR_INVALID);
  CHECK(jf_decode_attn_q4(&L, &pool, p, 1, 32, ip, 4, ip, NAN, 8, p, ws, p, nullptr) == JF_ERR_INVALID);
  CHECK(jf_decode_attn_q4(&L, &pool, p, 1, 32, ip, 4, ip, 1.0f, 8, p, ws, p, nullptr) == JF_OK);
  CHECK(jf_verify_attn_q4(&L, &pool, p, 1, 5, 32, ip, 4, ip, 1.0f, 8, p, ws, p, nullptr) == JF_ERR_UNSUPPORTED);
  // three tokens per request need three times the workspace of one
  CHECK(jf_verify_attn_q4(&L, &pool, p, 1, 3, 32, ip, 4, ip, 1.0f, 8, p, ws, p, nullptr) == JF_ERR_INVALID);
  CHECK(jf_verify_attn_q4(&L, &pool, p, 1, 3, 32, ip, 4, ip, 1.0f, 8, p, 3 * ws, p, nullptr) == JF_OK);
  CHECK(jf_prefill_attn_q4(&L, &pool, p, p, p, 16, 32, ip, 4, 4 * 256 + 1, 1.0f, p, nullptr) == JF_ERR_INVALID);
  CHECK(jf_reconstruct_q4(&L, &pool, ip, 4, 100, 7, 2, p, p, nullptr) == JF_ERR_INVALID);
  CHECK(jf_reconstruct_q4(&L, &pool, ip, 4, 100, 6, 2, p, p, nullptr) == JF_OK);
  jf_kv_layout bad = {256, 8, 96, 32, 16};
  size_t cb = 0, mb = 0;
  CHECK(jf_kv_pool_bytes(&bad, &cb, &mb) == JF_ERR_UNSUPPORTED);
  CHECK(jf_kv_pool_bytes(&L, &cb, &mb) == JF_OK && 2 * (cb + mb) == (size_t)16 * 256 * 1152);
  jf_kv_layout t4 = {256, 4, 256, 64, 16};
  CHECK(jf_tq4_pool_bytes(&L, &cb, &mb) == JF_ERR_UNSUPPORTED);
  CHECK(jf_tq4_pool_bytes(&t4, &cb, &mb) == JF_OK && cb == (size_t)16 * 4 * 256 * 128);
  const float* fp = reinterpret_cast<const float*>(p);
  CHECK(jf_tq4_decode_attn(&t4, p, p, p, p, fp, fp, fp, p, 1, 68, ip, 4, ip, 1.0f, 8, p, ws, p, nullptr) == JF_ERR_UNSUPPORTED);
  CHECK(jf_tq4_reconstruct(&t4, p, p, p, p, fp, fp, fp, ip, 4, 0, 0, 4, p, p, nullptr) == JF_OK);
  CHECK(jf_decode_step_q4_static(&L, &pool, p, p, p, 64, 32, ip, 4, ip, 1.0f, 64, p, nullptr) == JF_ERR_INVALID);
  CHECK(std::strlen(jf_version()) > 0);
}

// Snapshot save and restore through the CPU page-run copy: bytes round-trip
// into other pages, and malformed files, tables and buffers are refused.
static void snapshots() {
  jf_kv_layout L = {64, 2, 128, 64, 20};
  size_t cb = 0, mb = 0, pb = 0;
  CHECK(jf_kv_pool_bytes(&L, &cb, &mb) == JF_OK);
  CHECK(jf_kv_page_bytes(&L, &pb) == JF_OK && pb == 2 * (cb + mb) / 20);
  const int n_layers = 3;
  std::vector<std::vector<uint8_t>> src, dst;
  std::mt19937 rng(3);
  std::vector<jf_kv_pool_ptrs> sp(n_layers), dp(n_layers);
  for (int l = 0; l < n_layers; ++l) {
    src.emplace_back(2 * (cb + mb) + 64);
    dst.emplace_back(2 * (cb + mb) + 64, 0xA5);
    for (auto& b : src.back()) b = (uint8_t)rng();
    // 16-byte aligned pieces: codes, meta of K then V
    auto carve = [&](std::vector<uint8_t>& v, jf_kv_pool_ptrs& pp) {
      uint8_t* base = reinterpret_cast<uint8_t*>(((uintptr_t)v.data() + 15) & ~(uintptr_t)15);
      pp = {base, base + cb, base + cb + mb, base + 2 * cb + mb};
      stub_register(base, 2 * (cb + mb), true);
    };
    carve(src.back(), sp[l]);
    carve(dst.back(), dp[l]);
  }
  const int32_t n_pos = 64 * 7 + 13, n_pages = 8, max_pages = 9;
  std::vector<int32_t> t1 = {3, 17, 0, 5, 9, 11, 2, 19, -1}, t2 = {1, 4, 6, 8, 10, 12, 13, 14, -1};
  stub_register(t1.data(), t1.size() * 4, true);
  stub_register(t2.data(), t2.size() * 4, true);
  const size_t stage = 5 * pb;  // two halves of two pages (one page left over)
  std::vector<uint8_t> sd(stage + 16), sh(stage + 16);
  uint8_t* sdp = reinterpret_cast<uint8_t*>(((uintptr_t)sd.data() + 15) & ~(uintptr_t)15);
  uint8_t* shp = reinterpret_cast<uint8_t*>(((uintptr_t)sh.data() + 15) & ~(uintptr_t)15);
  stub_register(sdp, stage, true);
  stub_register(shp, stage, false);
  char dir[] = "/tmp/jfkv_sanXXXXXX";
  CHECK(mkdtemp(dir) != nullptr);
  const std::string path = std::string(dir) + "/s.safetensors";
  CHECK(jf_snapshot_save(path.c_str(), &L, sp.data(), n_layers, t1.data(), t1.data(), max_pages,
                         n_pos, sdp, shp, stage, nullptr) == JF_OK);
  CHECK(access((path + ".tmp").c_str(), F_OK) != 0);
  int32_t got = -1;
  CHECK(jf_snapshot_restore(path.c_str(), &L, dp.data(), n_layers, t2.data(), t2.data(),
                            max_pages, sdp, shp, stage, &got, nullptr) == JF_OK);
  CHECK(got == n_pos);
  const size_t sizes[4] = {cb / 20, mb / 20, cb / 20, mb / 20};
  for (int l = 0; l < n_layers; ++l)
    for (int i = 0; i < n_pages; ++i) {
      const uint8_t* a[4] = {(const uint8_t*)sp[l].k_codes, (const uint8_t*)sp[l].k_meta,
                             (const uint8_t*)sp[l].v_codes, (const uint8_t*)sp[l].v_meta};
      const uint8_t* b[4] = {(const uint8_t*)dp[l].k_codes, (const uint8_t*)dp[l].k_meta,
                             (const uint8_t*)dp[l].v_codes, (const uint8_t*)dp[l].v_meta};
      for (int r = 0; r < 4; ++r)
        CHECK(std::memcmp(a[r] + t1[i] * sizes[r], b[r] + t2[i] * sizes[r], sizes[r]) == 0);
    }
  // refusals
  CHECK(jf_snapshot_save(path.c_str(), &L, sp.data(), n_layers, t1.data(), t1.data(), max_pages,
                         n_pos, sdp, shp, pb, nullptr) == JF_ERR_INVALID);  // staging < 2 pages
  CHECK(jf_snapshot_save(path.c_str(), &L, sp.data(), n_layers, t1.data(), t1.data(), max_pages,
                         n_pos, shp, shp, stage, nullptr) == JF_ERR_INVALID);  // host as device
  CHECK(jf_snapshot_save((std::string(dir) + "/no/x").c_str(), &L, sp.data(), n_layers, t1.data(),
                         t1.data(), max_pages, n_pos, sdp, shp, stage, nullptr) == JF_ERR_IO);
  std::vector<int32_t> dup = {1, 4, 6, 8, 1, 12, 13, 14, -1};
  CHECK(jf_snapshot_restore(path.c_str(), &L, dp.data(), n_layers, dup.data(), dup.data(),
                            max_pages, sdp, shp, stage, &got, nullptr) == JF_ERR_INVALID);
  CHECK(jf_snapshot_restore(path.c_str(), &L, dp.data(), 2, t2.data(), t2.data(), max_pages, sdp,
                            shp, stage, &got, nullptr) == JF_ERR_INVALID);  // layer count
  // a truncated copy
  const std::string cut = std::string(dir) + "/cut.safetensors";
  {
    FILE* f = std::fopen(path.c_str(), "rb");
    std::vector<char> all(1 << 24);
    const size_t n = std::fread(all.data(), 1, all.size(), f);
    std::fclose(f);
    FILE* g = std::fopen(cut.c_str(), "wb");
    std::fwrite(all.data(), 1, n - 1, g);
    std::fclose(g);
  }
  CHECK(jf_snapshot_restore(cut.c_str(), &L, dp.data(), n_layers, t2.data(), t2.data(),
                            max_pages, sdp, shp, stage, &got, nullptr) == JF_ERR_INVALID);
  CHECK(jf_snapshot_restore((std::string(dir) + "/missing").c_str(), &L, dp.data(), n_layers,
                            t2.data(), t2.data(), max_pages, sdp, shp, stage, &got,
                            nullptr) == JF_ERR_IO);
  unlink(path.c_str());
  unlink(cut.c_str());
  rmdir(dir);
  stub_clear();
}

int main() {
  page_table_fuzz();
  validation();
  snapshots();
  std::printf("host driver: %d checks passed\n", g_checks);
  return 0;
}
