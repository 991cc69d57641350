// Split-K single-query decode attention over the paged 4-bit KV cache
// (gfx950, VALU; no matrix cores: one query row per head is not a dense
// contraction).
//
// The decode kernel reads the compressed pages where they are used instead of
// expanding the cache (Sec. 3.1, "Decode and prefill need different
// kernels"); heads are independent and query heads share their KV head
// (eq. groupattention).  Work is split over page-aligned ranges of each
// request ("split-K"); each split writes an fp32 partial (o, m, l) and the
// last split of a (request, KV head) to finish merges them with a
// log-sum-exp combine, so the workspace is bounded by the split cap, not by
// the context length.
//
// Data movement: every wave owns whole pages of its block's range and streams
// them row by row (a row = 32 positions at d = 128) through a private
// three-stage LDS ring filled by global_load_lds_dwordx4 (HBM -> LDS without
// registers), so two rows are always in flight while the third is consumed.
// K and V code rows are contiguous 2 KiB runs of a page; the (scale, bias)
// words are gathered transposed ([group][position]) so a lane reads both
// positions of its pair with one 8-byte LDS read.
//
// Mapping (d = 128): a "unit" of D/32 lanes owns a pair of adjacent
// positions; lane j of the unit holds dims 32j..32j+31 and reads 16 bytes of
// K codes per position and 32 bytes of position-paired V codes.
//
// Arithmetic: a 4-bit code masked into the low bits of an fp16 half is the
// subnormal c * 2^-24 (nibble at bits 4..7: 16c * 2^-24), which v_dot2
// multiplies exactly, so one AND per code pair replaces any conversion; the
// 2^24 (or 2^20) factor is folded into the fp32 scale afterwards.
//   - QK: pairs (dim 8m+k, dim 8m+k+4) of one position against the matching
//     fp16 query pairs (divided by 16 for the nibbles at bits 4..7); logit =
//     2^24 scale_g (q . c) + bias_g sum(q), summed over the unit's lanes;
//   - PV: the position-paired V layout gives (position 2s, position 2s+1) of
//     one dim per masked half-word pair, so v_dot2 against (w_2s, w_2s+1),
//     w = p * scale (fp16), accumulates both positions at once; the bias part
//     is sum(p * bias) per group, added once at the end.
// Online softmax keeps one running maximum per head per wave; it is raised
// only when a logit exceeds it by more than 2 (log2 units), so p <= 4 and
// p * scale stays within fp16 for any fp16 scale, and rescaling is rare.
#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>

#include "jfkv_internal.h"

namespace {

typedef _Float16 h2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) void lds_void;

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kTau = 2.0f;   // lazy-rescale margin, log2 units
// Initial running maximum: finite, so that a row with every position masked
// (-inf logits) before any valid one gives p = 2^(-inf - kMinit) = 0, not NaN.
constexpr float kMinit = -1e30f;
constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;
constexpr int kCodeBytes = 4096;  // K + V codes of one row (any supported d)
constexpr int kRingBudget = 73728;  // LDS bytes per block for the rings (2 blocks per CU)

__device__ __forceinline__ h2 as_h2(uint32_t u) { return __builtin_bit_cast(h2, u); }
__device__ __forceinline__ uint32_t as_u32(h2 v) { return __builtin_bit_cast(uint32_t, v); }
__device__ __forceinline__ float dot2(uint32_t a, h2 b, float c) {
  return __builtin_amdgcn_fdot2(as_h2(a), b, c, false);
}
__device__ __forceinline__ float dot2h(h2 a, uint32_t b, float c) {
  return __builtin_amdgcn_fdot2(a, as_h2(b), c, false);
}
__device__ __forceinline__ float lo_f(uint32_t u) { return (float)as_h2(u).x; }
__device__ __forceinline__ float hi_f(uint32_t u) { return (float)as_h2(u).y; }

// Cross-lane sums within aligned groups of 2, 4 or 8 lanes (DPP).
__device__ __forceinline__ float dpp_f(float v, int ctrl) {
  switch (ctrl) {  // the control must be an immediate
    case 0xB1:
      return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v),
                                                                   0xB1, 0xF, 0xF, true));
    case 0x4E:
      return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v),
                                                                   0x4E, 0xF, 0xF, true));
    default:  // 0x141: mirror within each half-row of 8 lanes
      return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v),
                                                                   0x141, 0xF, 0xF, true));
  }
}
template <int LPP>
__device__ __forceinline__ float unit_sum(float v) {
  if (LPP >= 2) v += dpp_f(v, 0xB1);   // lane ^ 1
  if (LPP >= 4) v += dpp_f(v, 0x4E);   // lane ^ 2
  if (LPP >= 8) v += dpp_f(v, 0x141);  // 7 - lane within 8
  return v;
}

// Value of lane h of each unit (LPP lanes), for every lane of the unit.
template <int LPP>
__device__ __forceinline__ uint32_t bcast_head_u(uint32_t v, int h) {
  const int x = (int)v;
  if constexpr (LPP == 4) {
    switch (h) {
      case 0: return (uint32_t)__builtin_amdgcn_update_dpp(0, x, 0x00, 0xF, 0xF, false);
      case 1: return (uint32_t)__builtin_amdgcn_update_dpp(0, x, 0x55, 0xF, 0xF, false);
      case 2: return (uint32_t)__builtin_amdgcn_update_dpp(0, x, 0xAA, 0xF, 0xF, false);
      default: return (uint32_t)__builtin_amdgcn_update_dpp(0, x, 0xFF, 0xF, 0xF, false);
    }
  } else {  // LPP == 2: quad_perm [h, h, 2+h, 2+h]
    if (h == 0) return (uint32_t)__builtin_amdgcn_update_dpp(0, x, 0xA0, 0xF, 0xF, false);
    return (uint32_t)__builtin_amdgcn_update_dpp(0, x, 0xF5, 0xF, 0xF, false);
  }
}
template <int LPP>
__device__ __forceinline__ float bcast_head(float v, int h) {
  return __builtin_bit_cast(float, bcast_head_u<LPP>(__builtin_bit_cast(uint32_t, v), h));
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) v = fmaxf(v, __shfl_xor(v, off));
  return v;
}
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) v += __shfl_xor(v, off);
  return v;
}

__device__ __forceinline__ void dma16(const void* g, void* lds_base) {
  __builtin_amdgcn_global_load_lds(g, (lds_void*)lds_base, 16, 0, 0);
}
__device__ __forceinline__ void dma4(const void* g, void* lds_base) {
  __builtin_amdgcn_global_load_lds(g, (lds_void*)lds_base, 4, 0, 0);
}

// Wait until at most N vector-memory operations of this wave are in flight.
template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

// Reads of the staged data of one position pair, issued together and waited
// for once: the two 16-byte K runs and the (t0, t1) meta words of the lane's
// group for K and V; later the 32 bytes of position-paired V codes.
// (Written as asm: the compiler would otherwise treat every LDS read as
// dependent on all outstanding LDS-DMA loads and serialize the ring.)
__device__ __forceinline__ void lds_read_k(uint32_t k0_addr, uint32_t k1_addr, uint32_t km_addr,
                                           uint32_t vm_addr, uint4& k0, uint4& k1, uint2& km,
                                           uint2& vm) {
  asm volatile(
      "ds_read_b128 %0, %4\n\t"
      "ds_read_b128 %1, %5\n\t"
      "ds_read_b64 %2, %6\n\t"
      "ds_read_b64 %3, %7\n\t"
      "s_waitcnt lgkmcnt(0)"
      : "=&v"(k0), "=&v"(k1), "=&v"(km), "=&v"(vm)
      : "v"(k0_addr), "v"(k1_addr), "v"(km_addr), "v"(vm_addr)
      : "memory");
}
__device__ __forceinline__ void lds_read_kv(uint32_t k0_addr, uint32_t k1_addr, uint32_t km_addr,
                                            uint32_t vm_addr, uint32_t v_addr, uint4& k0,
                                            uint4& k1, uint2& km, uint2& vm, uint4& v0,
                                            uint4& v1) {
  asm volatile(
      "ds_read_b128 %0, %6\n\t"
      "ds_read_b128 %1, %7\n\t"
      "ds_read_b64 %2, %8\n\t"
      "ds_read_b64 %3, %9\n\t"
      "ds_read_b128 %4, %10\n\t"
      "ds_read_b128 %5, %10 offset:16\n\t"
      "s_waitcnt lgkmcnt(0)"
      : "=&v"(k0), "=&v"(k1), "=&v"(km), "=&v"(vm), "=&v"(v0), "=&v"(v1)
      : "v"(k0_addr), "v"(k1_addr), "v"(km_addr), "v"(vm_addr), "v"(v_addr)
      : "memory");
}
__device__ __forceinline__ void lds_read_v(uint32_t v_addr, uint4& v0, uint4& v1) {
  asm volatile(
      "ds_read_b128 %0, %2\n\t"
      "ds_read_b128 %1, %2 offset:16\n\t"
      "s_waitcnt lgkmcnt(0)"
      : "=&v"(v0), "=&v"(v1)
      : "v"(v_addr)
      : "memory");
}

// Page-aligned split s of n_pages pages into S parts (remainder first).
__device__ __forceinline__ void split_range(int n_pages, int S, int s, int& pb, int& pe) {
  const int base = n_pages / S, rem = n_pages % S;
  pb = s * base + min(s, rem);
  pe = pb + base + (s < rem ? 1 : 0);
}

template <int D, int G, int HPB>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2))) void decode_kernel(
    const uint8_t* __restrict__ k_codes, const uint32_t* __restrict__ k_meta,
    const uint8_t* __restrict__ v_codes, const uint32_t* __restrict__ v_meta,
    const __half* __restrict__ q, const int32_t* __restrict__ block_tables,
    const int32_t* __restrict__ seq_lens, float* __restrict__ ws, int Hq, int Hkv, int P, int NP,
    int max_pages, int max_splits, int n_hchunks, float scale_log2) {
  constexpr int LPP = D / 32;            // lanes per position pair (unit)
  constexpr int UNITS = 64 / LPP;        // units per wave
  constexpr int ROWPOS = 2 * UNITS;      // positions per row
  constexpr int NG = D / G;              // scale groups per head
  constexpr int META_WORDS = ROWPOS * NG;          // per row, K or V
  constexpr int META_DMAS = (META_WORDS + 63) / 64;
  constexpr int DMAS_PER_ROW = 4 + 2 * META_DMAS;  // K 2, V 2, meta
  constexpr int kMetaBytes = 2 * 256 * META_DMAS;  // K then V meta, 256 B per DMA
  constexpr int kStageBytes = kCodeBytes + kMetaBytes;
  constexpr int kStages = kRingBudget / (kWaves * kStageBytes) >= 4 ? 4 : 3;
  static_assert(kStages <= 4, "wait cascade covers up to 3 rows ahead");
  // lane j of a unit owns head j's softmax state when there is one head per lane
  constexpr bool kLaneHeads = (LPP == HPB) && (LPP == 2 || LPP == 4);
  static_assert(ROWPOS * D == kCodeBytes, "row codes");
  static_assert(kStages * kWaves * kStageBytes <= kRingBudget, "ring size");

  __shared__ __attribute__((aligned(16))) uint8_t smem[kWaves][kStages][kStageBytes];

  const int split = blockIdx.x;
  const int kv = blockIdx.y / n_hchunks;
  const int hc = blockIdx.y % n_hchunks;
  const int b = blockIdx.z;
  const int gq = Hq / Hkv;
  const int h0 = kv * gq + hc * HPB;
  const int nh = min(HPB, gq - hc * HPB);
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform (scalar)

  const int L = min(seq_lens[b], max_pages * P);
  if (L <= 0) return;  // the combine writes the all-zero output row
  const int n_pages = (L + P - 1) / P;
  const int S = min(max_splits, n_pages);
  if (split >= S) return;
  int pb, pe;
  split_range(n_pages, S, split, pb, pe);
  const int t_end = min(pe * P, L);
  const int rows_per_page = P / ROWPOS;

  const int unit = lane / LPP;
  const int j = lane % LPP;
  const int g = (32 * j) / G;  // the lane's scale group

  // ---- query pairs in unpack order: word m (dims 8m..8m+7 of the lane's 32),
  // pair k = (dim 8m+k, dim 8m+k+4); odd k pre-divided by 16
  h2 qp[HPB][4][4];
  float qsum[HPB];
#pragma unroll
  for (int h = 0; h < HPB; ++h) {
    const int head = h0 + min(h, nh - 1);
    const uint4* src = reinterpret_cast<const uint4*>(q + ((size_t)b * Hq + head) * D + 32 * j);
    float s = 0.0f;
#pragma unroll
    for (int m = 0; m < 4; ++m) {
      const uint4 u = src[m];
      const uint32_t wq[4] = {u.x, u.y, u.z, u.w};
      _Float16 e[8];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        e[2 * i] = as_h2(wq[i]).x;
        e[2 * i + 1] = as_h2(wq[i]).y;
      }
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        const _Float16 f = (k & 1) ? (_Float16)0.0625f : (_Float16)1.0f;
        qp[h][m][k] = h2{e[k] * f, e[k + 4] * f};
        s += (float)e[k] + (float)e[k + 4];
      }
    }
    qsum[h] = s * scale_log2;
  }
  // logit (log2 units) = kscale * raw_dot + bias * qsum
  const float kfold = 16777216.0f * scale_log2;  // 2^24

  float m_mine = kMinit, thr_mine = kMinit, l_mine = 0.0f;  // head j (kLaneHeads)
  float m_run[HPB], l_acc[HPB], b_acc[HPB];
  float acc[HPB][32];
#pragma unroll
  for (int h = 0; h < HPB; ++h) {
    m_run[h] = kMinit;
    l_acc[h] = 0.0f;
    b_acc[h] = 0.0f;
#pragma unroll
    for (int i = 0; i < 32; ++i) acc[h][i] = 0.0f;
  }

  // ---- this wave's rows: pages pb + wave, pb + wave + 4, ...; every row of each
  const int my_pages = (pe - pb - wave + kWaves - 1) / kWaves;
  const int my_rows = (pe - pb > wave) ? my_pages * rows_per_page : 0;
  const size_t head_codes = (size_t)P * (D / 2);
  const size_t page_codes = (size_t)Hkv * head_codes;
  uint8_t* ring = smem[wave][0];
  const uint32_t ring_lds = (uint32_t)(uintptr_t)ring;

  // This wave's page IDs, 64 per vector register (lane k holds its k-th page of
  // the group), read per row with v_readlane: no memory access on the row path.
  auto load_group = [&](int grp) {
    const int k = 64 * grp + lane;
    return (k < my_pages) ? block_tables[(size_t)b * max_pages + pb + wave + k * kWaves] : -1;
  };
  int pg_cur = load_group(0), pg_nxt = load_group(1);
  int grp_cur = 0;
  auto page_of = [&](int pk) {  // pk: the wave's page index, within groups cur or cur+1
    const int g2 = pk >> 6;
    const int v = (g2 == grp_cur) ? __builtin_amdgcn_readlane(pg_cur, pk & 63)
                                  : __builtin_amdgcn_readlane(pg_nxt, pk & 63);
    return v;
  };

  // Issue the loads of row r (of this wave) into stage r % kStages.
  auto issue_row = [&](int r) {
    const int s0 = (r % rows_per_page) * ROWPOS;
    int page = page_of(r / rows_per_page);
    if ((unsigned)page >= (unsigned)NP) page = 0;  // never read past the pool; masked below
    uint8_t* st = ring + (r % kStages) * kStageBytes;
    const uint8_t* kc = k_codes + page * page_codes + kv * head_codes + (size_t)s0 * (D / 2);
    const uint8_t* vc = v_codes + page * page_codes + kv * head_codes + (size_t)(s0 / 2) * D;
    dma16(kc + 16 * lane, st);
    dma16(kc + 1024 + 16 * lane, st + 1024);
    dma16(vc + 16 * lane, st + 2048);
    dma16(vc + 1024 + 16 * lane, st + 3072);
    const size_t mbase = (((size_t)page * Hkv + kv) * P + s0) * NG;
#pragma unroll
    for (int i = 0; i < META_DMAS; ++i) {
      const int w = 64 * i + lane;  // transposed: word w = (group w / ROWPOS, pos w % ROWPOS)
      const int wi = (w < META_WORDS) ? w : 0;
      const size_t src = mbase + (size_t)(wi % ROWPOS) * NG + wi / ROWPOS;
      if (w < META_WORDS) {
        dma4(k_meta + src, st + kCodeBytes + 256 * i);
        dma4(v_meta + src, st + kCodeBytes + kMetaBytes / 2 + 256 * i);
      }
    }
  };

  for (int r = 0; r < kStages - 1 && r < my_rows; ++r) issue_row(r);

  const h2 ones = {(_Float16)1.0f, (_Float16)1.0f};
  for (int r = 0; r < my_rows; ++r) {
    // rows issued after row r: min(kStages - 1, my_rows - 1 - r); wait until
    // only those are in flight
    if (r + kStages - 1 < my_rows) issue_row(r + kStages - 1);
    const int ahead = min(kStages - 1, my_rows - 1 - r);
    if (ahead >= 3) {
      wait_vm<DMAS_PER_ROW * 3>();
    } else if (ahead == 2) {
      wait_vm<DMAS_PER_ROW * 2>();
    } else if (ahead == 1) {
      wait_vm<DMAS_PER_ROW>();
    } else {
      wait_vm<0>();
    }
    const int pk = r / rows_per_page;
    const int pi = pb + wave + pk * kWaves;
    const int page = page_of(pk);
    const int t_row = pi * P + (r % rows_per_page) * ROWPOS;
    if ((r % rows_per_page) == rows_per_page - 1 && ((pk + 1) & 63) == 0) {
      // leaving page group grp_cur: shift the groups (the ring already holds
      // rows of the next group, whose IDs come from pg_nxt)
      grp_cur += 1;
      pg_cur = pg_nxt;
      pg_nxt = load_group(grp_cur + 1);
    }
    const int t0 = t_row + 2 * unit;
    const bool pg_ok = (unsigned)page < (unsigned)NP;
    const bool ok0 = pg_ok && t0 < t_end, ok1 = pg_ok && t0 + 1 < t_end;

    const uint32_t st = ring_lds + (r % kStages) * kStageBytes;
    uint4 kw0, kw1, vw0, vw1;
    uint2 km, vm;
#ifdef JF_SPLIT_LDS_READS
    lds_read_k(st + (2 * unit) * (D / 2) + 16 * j, st + (2 * unit + 1) * (D / 2) + 16 * j,
               st + kCodeBytes + (g * ROWPOS + 2 * unit) * 4,
               st + kCodeBytes + kMetaBytes / 2 + (g * ROWPOS + 2 * unit) * 4, kw0, kw1, km, vm);
#else
    lds_read_kv(st + (2 * unit) * (D / 2) + 16 * j, st + (2 * unit + 1) * (D / 2) + 16 * j,
                st + kCodeBytes + (g * ROWPOS + 2 * unit) * 4,
                st + kCodeBytes + kMetaBytes / 2 + (g * ROWPOS + 2 * unit) * 4,
                st + 2048 + unit * D + 32 * j, kw0, kw1, km, vm, vw0, vw1);
#endif

    // ---- QK partial dot products over the lane's 32 dims
    float d0[HPB], d1[HPB];
#pragma unroll
    for (int h = 0; h < HPB; ++h) d0[h] = d1[h] = 0.0f;
    {
      const uint32_t ka[4] = {kw0.x, kw0.y, kw0.z, kw0.w};
      const uint32_t kb[4] = {kw1.x, kw1.y, kw1.z, kw1.w};
#pragma unroll
      for (int m = 0; m < 4; ++m) {
        const uint32_t a8 = ka[m] >> 8, b8 = kb[m] >> 8;
        const uint32_t ca[4] = {ka[m] & 0x000F000Fu, ka[m] & 0x00F000F0u, a8 & 0x000F000Fu,
                                a8 & 0x00F000F0u};
        const uint32_t cb[4] = {kb[m] & 0x000F000Fu, kb[m] & 0x00F000F0u, b8 & 0x000F000Fu,
                                b8 & 0x00F000F0u};
#pragma unroll
        for (int h = 0; h < HPB; ++h)
#pragma unroll
          for (int k = 0; k < 4; ++k) {
            d0[h] = dot2(ca[k], qp[h][m][k], d0[h]);
            d1[h] = dot2(cb[k], qp[h][m][k], d1[h]);
          }
      }
    }
    const float sk0 = lo_f(km.x) * kfold, bk0 = hi_f(km.x);
    const float sk1 = lo_f(km.y) * kfold, bk1 = hi_f(km.y);
    const bool full = pg_ok && t_row + ROWPOS <= t_end;  // wave-uniform
    float v0[HPB], v1[HPB];
#pragma unroll
    for (int h = 0; h < HPB; ++h) {
      v0[h] = fmaf(sk0, d0[h], bk0 * qsum[h]);
      v1[h] = fmaf(sk1, d1[h], bk1 * qsum[h]);
    }
    const uint32_t vm0 = ok0 ? vm.x : 0u, vm1 = ok1 ? vm.y : 0u;
    const h2 sv = as_h2(__builtin_amdgcn_perm(vm1, vm0, 0x05040100u));  // (s_t0, s_t1)
    const uint32_t bv = __builtin_amdgcn_perm(vm1, vm0, 0x07060302u);    // (b_t0, b_t1)
    h2 W[HPB];
    if constexpr (kLaneHeads) {
      // reduce-scatter over the unit: lane j keeps the full logits of head j
      float sm0, sm1;
      if constexpr (LPP == 4) {
        const bool odd = j & 1, hi = j & 2;
        float k00 = odd ? v0[1] : v0[0], k01 = odd ? v0[3] : v0[2];
        float k10 = odd ? v1[1] : v1[0], k11 = odd ? v1[3] : v1[2];
        const float s00 = odd ? v0[0] : v0[1], s01 = odd ? v0[2] : v0[3];
        const float s10 = odd ? v1[0] : v1[1], s11 = odd ? v1[2] : v1[3];
        k00 += dpp_f(s00, 0xB1);
        k01 += dpp_f(s01, 0xB1);
        k10 += dpp_f(s10, 0xB1);
        k11 += dpp_f(s11, 0xB1);
        sm0 = (hi ? k01 : k00) + dpp_f(hi ? k00 : k01, 0x4E);
        sm1 = (hi ? k11 : k10) + dpp_f(hi ? k10 : k11, 0x4E);
      } else {  // LPP == 2
        const bool odd = j & 1;
        sm0 = (odd ? v0[1] : v0[0]) + dpp_f(odd ? v0[0] : v0[1], 0xB1);
        sm1 = (odd ? v1[1] : v1[0]) + dpp_f(odd ? v1[0] : v1[1], 0xB1);
      }
      if (!full) {
        sm0 = ok0 ? sm0 : -INFINITY;
        sm1 = ok1 ? sm1 : -INFINITY;
      }
      if (__builtin_amdgcn_ballot_w64(fmaxf(sm0, sm1) > thr_mine) != 0) {
        float mx = fmaxf(sm0, sm1);
#pragma unroll
        for (int off = LPP; off < 64; off <<= 1) mx = fmaxf(mx, __shfl_xor(mx, off));
        float alpha = 1.0f;
        if (mx > m_mine) {  // uniform across the lanes of head j
          alpha = __builtin_amdgcn_exp2f(m_mine - mx);
          m_mine = mx;
          thr_mine = mx + kTau;
        }
        l_mine *= alpha;
#pragma unroll
        for (int h = 0; h < HPB; ++h) {
          const float ah = bcast_head<LPP>(alpha, h);
          b_acc[h] *= ah;
#pragma unroll
          for (int i = 0; i < 32; ++i) acc[h][i] *= ah;
        }
      }
      const float p0 = __builtin_amdgcn_exp2f(sm0 - m_mine);
      const float p1 = __builtin_amdgcn_exp2f(sm1 - m_mine);
      const h2 pm = h2{(_Float16)p0, (_Float16)p1};
      l_mine = __builtin_amdgcn_fdot2(pm, ones, l_mine, false);
#pragma unroll
      for (int h = 0; h < HPB; ++h) {
        const h2 ph = as_h2(bcast_head_u<LPP>(as_u32(pm), h));
        b_acc[h] = dot2h(ph, bv, b_acc[h]);
        W[h] = ph * sv;
      }
    } else {
      float s0[HPB], s1[HPB];
      bool need = false;
#pragma unroll
      for (int h = 0; h < HPB; ++h) {
        const float a = unit_sum<LPP>(v0[h]);
        const float c = unit_sum<LPP>(v1[h]);
        s0[h] = ok0 ? a : -INFINITY;
        s1[h] = ok1 ? c : -INFINITY;
        need |= fmaxf(s0[h], s1[h]) > m_run[h] + kTau;
      }
      if (__builtin_amdgcn_ballot_w64(need) != 0) {
#pragma unroll
        for (int h = 0; h < HPB; ++h) {
          const float mx = wave_max(fmaxf(s0[h], s1[h]));
          if (mx > m_run[h]) {  // wave-uniform
            const float alpha = __builtin_amdgcn_exp2f(m_run[h] - mx);
            m_run[h] = mx;
            l_acc[h] *= alpha;
            b_acc[h] *= alpha;
#pragma unroll
            for (int i = 0; i < 32; ++i) acc[h][i] *= alpha;
          }
        }
      }
#pragma unroll
      for (int h = 0; h < HPB; ++h) {
        const float p0 = __builtin_amdgcn_exp2f(s0[h] - m_run[h]);
        const float p1 = __builtin_amdgcn_exp2f(s1[h] - m_run[h]);
        const h2 pp = h2{(_Float16)p0, (_Float16)p1};
        l_acc[h] = __builtin_amdgcn_fdot2(pp, ones, l_acc[h], false);
        b_acc[h] = dot2h(pp, bv, b_acc[h]);
        W[h] = pp * sv;
      }
    }
#ifdef JF_SPLIT_LDS_READS
    lds_read_v(st + 2048 + unit * D + 32 * j, vw0, vw1);
#endif
    const uint32_t va[8] = {vw0.x, vw0.y, vw0.z, vw0.w, vw1.x, vw1.y, vw1.z, vw1.w};
#pragma unroll
    for (int m = 0; m < 8; ++m) {
      const uint32_t w8 = va[m] >> 8;
      const uint32_t c[4] = {va[m] & 0x000F000Fu, va[m] & 0x00F000F0u, w8 & 0x000F000Fu,
                             w8 & 0x00F000F0u};  // (dim 4m+k of t0, of t1)
#pragma unroll
      for (int h = 0; h < HPB; ++h)
#pragma unroll
        for (int k = 0; k < 4; ++k)
          acc[h][4 * m + k] = __builtin_amdgcn_fdot2(W[h], as_h2(c[k]), acc[h][4 * m + k], false);
    }
  }
  wait_vm<0>();
  if constexpr (kLaneHeads) {
#pragma unroll
    for (int h = 0; h < HPB; ++h) {
      m_run[h] = bcast_head<LPP>(m_mine, h);
      l_acc[h] = bcast_head<LPP>(l_mine, h);
    }
  }
  __syncthreads();  // all waves done with their rings: reuse LDS for the merge

  // ---- merge the units of each wave and the waves of the block
  float* red = reinterpret_cast<float*>(&smem[0][0][0]);  // [kWaves][UNITS][D]
  float* red_l = red + kWaves * UNITS * D;                // [kWaves][UNITS]
  float* red_m = red_l + kWaves * UNITS;                  // [kWaves][HPB]
  static_assert(sizeof(float) * (kWaves * UNITS * (D + 1) + kWaves * HPB) <=
                    sizeof(smem), "merge buffer");
  if (lane == 0) {
#pragma unroll
    for (int h = 0; h < HPB; ++h) red_m[wave * HPB + h] = m_run[h];
  }
  __syncthreads();
  const int n_rec = Hq * max_splits;
#pragma unroll
  for (int h = 0; h < HPB; ++h) {
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) M = fmaxf(M, red_m[w * HPB + h]);
    const float f = (m_run[h] == -INFINITY) ? 0.0f : __builtin_amdgcn_exp2f(m_run[h] - M);
#pragma unroll
    for (int i = 0; i < 32; ++i) {
      // undo the 2^-24 (even dims) or 2^-20 (odd dims of each 4) code factor
      const float cf = (i & 1) ? 1048576.0f : 16777216.0f;
      red[(wave * UNITS + unit) * D + 32 * j + i] = fmaf(acc[h][i], cf, b_acc[h]) * f;
    }
    if (j == 0) red_l[wave * UNITS + unit] = l_acc[h] * f;
    __syncthreads();
    if (h < nh) {
      for (int i = tid; i < D; i += kThreads) {
        float o4[8] = {0, 0, 0, 0, 0, 0, 0, 0}, l4[8] = {0, 0, 0, 0, 0, 0, 0, 0};
#pragma unroll
        for (int u = 0; u < kWaves * UNITS; ++u) {  // independent partial sums
          o4[u & 7] += red[u * D + i];
          l4[u & 7] += red_l[u];
        }
        float o = 0.0f, l = 0.0f;
#pragma unroll
        for (int k = 0; k < 8; ++k) {
          o += o4[k];
          l += l4[k];
        }
        float* rec = ws + (((size_t)b * Hq + (h0 + h)) * max_splits + split) * (D + 2);
        rec[i] = (l > 0.0f) ? o / l : 0.0f;
        if (i == 0) {
          rec[D] = M;
          rec[D + 1] = l;
        }
      }
    }
    __syncthreads();
  }
  (void)n_rec;

}

// Log-sum-exp combine of a (request, query head)'s split partials (a
// separate kernel: the kernel boundary makes every split's partial visible,
// while an in-kernel ticket would need device-scope fences, which write back
// an XCD's L2 on this GPU).  256 threads: 256/D threads per dim, each summing
// a strided subset of the splits with independent loads.
constexpr int kCombineThreads = 512;

template <int D>
__global__ __launch_bounds__(kCombineThreads) void decode_combine_kernel(
    const float* __restrict__ ws, const int32_t* __restrict__ seq_lens, __half* __restrict__ out,
    int Hq, int P, int max_pages, int max_splits) {
  constexpr int NT = kCombineThreads, NW = NT / 64;
  constexpr int PARTS = NT / D;
  __shared__ float s_w[1024];
  __shared__ float s_red[NW];
  __shared__ float s_part[PARTS][D];
  const int h = blockIdx.x, b = blockIdx.y, tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int L = min(seq_lens[b], max_pages * P);
  __half* dst = out + ((size_t)b * Hq + h) * D;
  if (L <= 0) {
    if (tid < D) dst[tid] = __float2half(0.0f);
    return;
  }
  const int n_pages = (L + P - 1) / P;
  const int S = min(max_splits, n_pages);
  const float* recs = ws + ((size_t)b * Hq + h) * max_splits * (D + 2);
  // one round of loads for every split's (m, l); S <= 1024
  float mv[2], lv[2];
  float M = -INFINITY;
#pragma unroll
  for (int k = 0; k < 2; ++k) {
    const int s = tid + k * NT;
    mv[k] = (s < S) ? recs[(size_t)s * (D + 2) + D] : -INFINITY;
    lv[k] = (s < S) ? recs[(size_t)s * (D + 2) + D + 1] : 0.0f;
    M = fmaxf(M, mv[k]);
  }
  M = wave_max(M);
  if (lane == 0) s_red[wave] = M;
  __syncthreads();
  M = s_red[0];
#pragma unroll
  for (int w = 1; w < NW; ++w) M = fmaxf(M, s_red[w]);
  float den = 0.0f;
#pragma unroll
  for (int k = 0; k < 2; ++k) {
    const int s = tid + k * NT;
    const float w = (s < S && mv[k] != -INFINITY) ? lv[k] * __builtin_amdgcn_exp2f(mv[k] - M) : 0.0f;
    if (s < S) s_w[s] = w;
    den += w;
  }
  den = wave_sum(den);
  __syncthreads();  // s_red reads done before it is reused
  if (lane == 0) s_red[wave] = den;
  __syncthreads();
  den = 0.0f;
#pragma unroll
  for (int w = 0; w < NW; ++w) den += s_red[w];
  // weighted sum: thread (part, dim) takes splits part, part+PARTS, ...; 16
  // independent loads per round
  const int i = tid % D, part = tid / D;
  float acc[16];
#pragma unroll
  for (int k = 0; k < 16; ++k) acc[k] = 0.0f;
  for (int s0 = part; s0 < S; s0 += 16 * PARTS) {
#pragma unroll
    for (int k = 0; k < 16; ++k) {
      const int s = s0 + k * PARTS;
      if (s < S) acc[k] = fmaf(s_w[s], recs[(size_t)s * (D + 2) + i], acc[k]);
    }
  }
  float num = 0.0f;
#pragma unroll
  for (int k = 0; k < 16; ++k) num += acc[k];
  s_part[part][i] = num;
  __syncthreads();
  if (tid < D) {
    float o = 0.0f;
#pragma unroll
    for (int k = 0; k < PARTS; ++k) o += s_part[k][tid];
    dst[tid] = __float2half_rn((den > 0.0f && M != -INFINITY) ? o / den : 0.0f);
  }
}

template <int D, int G, int HPB>
hipError_t launch_t(const jf_kv_layout& L, const jf_kv_pool_ptrs& pool, const void* q,
                    int32_t B, int32_t Hq, const int32_t* bt, int32_t max_pages,
                    const int32_t* lens, float scale, int32_t max_splits, void* ws, void* out,
                    hipStream_t stream) {
  const int gq = Hq / L.num_kv_heads;
  const int n_hchunks = (gq + HPB - 1) / HPB;
  dim3 grid(max_splits, L.num_kv_heads * n_hchunks, B);
  hipLaunchKernelGGL((decode_kernel<D, G, HPB>), grid, dim3(kThreads), 0, stream,
                     static_cast<const uint8_t*>(pool.k_codes),
                     static_cast<const uint32_t*>(pool.k_meta),
                     static_cast<const uint8_t*>(pool.v_codes),
                     static_cast<const uint32_t*>(pool.v_meta), static_cast<const __half*>(q),
                     bt, lens, static_cast<float*>(ws), Hq, L.num_kv_heads, L.page_size,
                     L.num_pages, max_pages, max_splits, n_hchunks, scale * kLog2e);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((decode_combine_kernel<D>), dim3(Hq, B), dim3(kCombineThreads), 0, stream,
                     static_cast<const float*>(ws), lens, static_cast<__half*>(out), Hq,
                     L.page_size, max_pages, max_splits);
  return hipGetLastError();
}

template <int D, int G>
hipError_t dispatch_hpb(const jf_kv_layout& L, const jf_kv_pool_ptrs& pool, const void* q,
                        int32_t B, int32_t Hq, const int32_t* bt, int32_t max_pages,
                        const int32_t* lens, float scale, int32_t max_splits, void* ws,
                        void* out, hipStream_t stream) {
  const int gq = Hq / L.num_kv_heads;
#define JF_ARGS L, pool, q, B, Hq, bt, max_pages, lens, scale, max_splits, ws, out, stream
  if (gq == 1) return launch_t<D, G, 1>(JF_ARGS);
  if (gq == 2) return launch_t<D, G, 2>(JF_ARGS);
  if (gq % 3 == 0 && gq % 4 != 0) return launch_t<D, G, 3>(JF_ARGS);
  return launch_t<D, G, 4>(JF_ARGS);
#undef JF_ARGS
}

}  // namespace

namespace jfkv {

hipError_t launch_decode(const jf_kv_layout& L, const jf_kv_pool_ptrs& pool, const void* q,
                         int32_t B, int32_t Hq, const int32_t* bt, int32_t max_pages,
                         const int32_t* lens, float scale, int32_t max_splits, void* ws,
                         void* out, hipStream_t stream) {
#define JF_ARGS L, pool, q, B, Hq, bt, max_pages, lens, scale, max_splits, ws, out, stream
#define JF_CASE(D_, G_) \
  if (L.head_dim == D_ && L.group_size == G_) return dispatch_hpb<D_, G_>(JF_ARGS);
  JF_CASE(64, 32)
  JF_CASE(64, 64)
  JF_CASE(128, 32)
  JF_CASE(128, 64)
  JF_CASE(128, 128)
  JF_CASE(256, 32)
  JF_CASE(256, 64)
  JF_CASE(256, 128)
#undef JF_CASE
#undef JF_ARGS
  return hipErrorInvalidValue;
}

}  // namespace jfkv
