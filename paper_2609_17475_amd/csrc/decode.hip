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

#include <type_traits>

#include "jfkv_internal.h"

namespace {

typedef _Float16 h2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) void lds_void;

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kTau = 2.0f;   // lazy-rescale margin, log2 units
// Initial running maximum: finite, so that a row with every position masked
// (-inf logits) before any valid one gives p = 2^(-inf - kMinit) = 0, not NaN.
constexpr float kMinit = -1e30f;
constexpr int kThreads = 256;     // 4 waves: one split; two blocks per CU
constexpr int kWaves = kThreads / 64;
constexpr int kSplitWaves = kWaves;  // waves per split
constexpr int kCodeBytes = 4096;  // K + V codes of one row (any supported d)
constexpr int kRingBudget = 81920;  // LDS bytes per block for the rings (half of a CU's LDS)

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

// First product of a dot-product chain: v_dot2 with a zero accumulator (the
// compiler would otherwise zero a register and accumulate into it).
__device__ __forceinline__ float dot2_first(uint32_t a, h2 b) {
  float d;
  asm("v_dot2_f32_f16 %0, %1, %2, 0" : "=v"(d) : "v"(a), "v"(b));
  return d;
}
// s * n + b * q with s and b the low and high fp16 halves of one (scale,
// bias) word, converted exactly inside v_fma_mix.
__device__ __forceinline__ float fold_meta(uint32_t sb, float n, float q) {
  float t, r;
  asm("v_fma_mix_f32 %0, %1, %2, 0 op_sel:[1,0,0] op_sel_hi:[1,0,0]" : "=v"(t) : "v"(sb), "v"(q));
  asm("v_fma_mix_f32 %0, %1, %2, %3 op_sel_hi:[1,0,0]" : "=v"(r) : "v"(sb), "v"(n), "v"(t));
  return r;
}

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

// Lane index from a volatile instruction: code that uses it cannot be hoisted
// out of a loop, so rarely taken paths keep no lane-derived registers live.
__device__ __forceinline__ int lane_id_volatile() {
  int l;
  asm volatile("v_mbcnt_lo_u32_b32 %0, -1, 0\n\tv_mbcnt_hi_u32_b32 %0, -1, %0" : "=v"(l));
  return l;
}
__device__ __forceinline__ float shfl_xor_at(float v, int lane, int off) {
  return __builtin_bit_cast(float,
                            __builtin_amdgcn_ds_bpermute((lane ^ off) << 2, __builtin_bit_cast(int, v)));
}
// Maximum over lanes lane % from .. == const: offsets from, 2 from, ..., 32.
__device__ __forceinline__ float xor_max_from(float v, int from) {
  const int ln = lane_id_volatile();
  for (int off = from; off < 64; off <<= 1) v = fmaxf(v, shfl_xor_at(v, ln, off));
  return v;
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
// All reads of one staged row at compile-time offsets from three per-lane
// bases (K codes, meta words, V codes), waited for once.
template <int OFF, int VM>
__device__ __forceinline__ void lds_read_row(uint32_t k0_addr, uint32_t k1_addr, uint32_t m_addr,
                                             uint32_t v0_addr, uint32_t v1_addr, uint4& k0,
                                             uint4& k1, uint2& km, uint2& vm, uint4& v0,
                                             uint4& v1) {
  static_assert(OFF >= 0 && OFF + VM < 65536, "ds offsets");
  asm volatile(
      "ds_read_b128 %0, %6 offset:%11\n\t"
      "ds_read_b128 %1, %7 offset:%11\n\t"
      "ds_read_b64 %2, %8 offset:%11\n\t"
      "ds_read_b64 %3, %8 offset:%12\n\t"
      "ds_read_b128 %4, %9 offset:%11\n\t"
      "ds_read_b128 %5, %10 offset:%11\n\t"
      "s_waitcnt lgkmcnt(0)"
      : "=&v"(k0), "=&v"(k1), "=&v"(km), "=&v"(vm), "=&v"(v0), "=&v"(v1)
      : "v"(k0_addr), "v"(k1_addr), "v"(m_addr), "v"(v0_addr), "v"(v1_addr), "i"(OFF),
        "i"(OFF + VM)
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

// Sum over the units of a 16-lane row (lanes of equal j = lane % LPP):
// rotations by LPP, 2 LPP, ... within the row.
template <int N>
__device__ __forceinline__ float row_ror_add(float v) {
  return v + __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v),
                                                                   0x120 + N, 0xF, 0xF, true));
}
template <int LPP>
__device__ __forceinline__ float row_units_sum(float v) {
  if constexpr (LPP <= 2) v = row_ror_add<2>(v);
  if constexpr (LPP <= 4) v = row_ror_add<4>(v);
  if constexpr (LPP <= 8) v = row_ror_add<8>(v);
  return v;
}

// Page-aligned split s of n_pages pages into S parts (remainder first).
__device__ __forceinline__ void split_range(int n_pages, int S, int s, int& pb, int& pe) {
  const int base = n_pages / S, rem = n_pages % S;
  pb = s * base + min(s, rem);
  pe = pb + base + (s < rem ? 1 : 0);
}

// Coherent (sc1: device-scope) buffer loads of split records; the resource
// covers one head's records, so every access is bounds-checked by the
// hardware as well.
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
constexpr int kCpolSc1 = 16;
__device__ __forceinline__ __amdgpu_buffer_rsrc_t records_rsrc(const float* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(base), (short)0, (int)bytes,
                                           0x00020000);
}

// Log-sum-exp combine of the split records of heads h0 .. h0+nh-1 (nh <= 4)
// of request b: M = max m_s, w_s = l_s 2^(m_s - M), o = sum w_s o_s / sum w_s.
// Wave w combines head w: lane (c, k) holds dims 4c..4c+3 and the splits
// s = k, k + KP, ... (KP = 64 / (D/4)), fetched KCH at a time with coherent
// loads and folded into a running maximum; the KP parts meet by shuffles.
// Records: [max_splits][D + 4] fp32 per head (o/l in 0..D-1, m at D, l at
// D+1).
template <int D>
__device__ void combine_splits(const float* ws, __half* out, int b, int Hq, int h0, int nh,
                               int max_splits, int S) {
  constexpr int CPL = D / 4;      // float4 chunks of a record's o
  constexpr int KP = 64 / CPL;    // lanes per chunk (split parts)
  constexpr int KCH = 8;          // splits per lane per round
  static_assert(KP >= 1 && 64 % CPL == 0, "");
  const int lane = threadIdx.x & 63, h = threadIdx.x >> 6;
  if (h >= nh) return;
  const int c = lane % CPL, k = lane / CPL;
  const float* recs = ws + ((size_t)b * Hq + h0 + h) * max_splits * (D + 4);
  const __amdgpu_buffer_rsrc_t rs = records_rsrc(recs, (uint32_t)S * (D + 4) * 4);
  float m_run = -INFINITY, den = 0.0f;
  float num[4] = {0.0f, 0.0f, 0.0f, 0.0f};
  for (int s0 = k; s0 < S; s0 += KP * KCH) {
    f32x4 o[KCH];
    f32x2 ml[KCH];
#pragma unroll
    for (int i = 0; i < KCH; ++i) {
      const int s = min(s0 + KP * i, S - 1);  // past the end: a valid record, weight 0
      o[i] = __builtin_amdgcn_raw_buffer_load_b128(rs, (s * (D + 4) + 4 * c) * 4, 0, kCpolSc1);
      ml[i] = __builtin_amdgcn_raw_buffer_load_b64(rs, (s * (D + 4) + D) * 4, 0, kCpolSc1);
    }
    float mx = m_run;
#pragma unroll
    for (int i = 0; i < KCH; ++i)
      if (s0 + KP * i < S && ml[i].y > 0.0f) mx = fmaxf(mx, ml[i].x);
    const float f = (m_run == -INFINITY) ? 0.0f : __builtin_amdgcn_exp2f(m_run - mx);
    den *= f;
#pragma unroll
    for (int e = 0; e < 4; ++e) num[e] *= f;
#pragma unroll
    for (int i = 0; i < KCH; ++i) {
      const bool on = s0 + KP * i < S && ml[i].y > 0.0f;
      const float w = on ? ml[i].y * __builtin_amdgcn_exp2f(ml[i].x - mx) : 0.0f;
      den += w;
      num[0] = fmaf(w, o[i].x, num[0]);
      num[1] = fmaf(w, o[i].y, num[1]);
      num[2] = fmaf(w, o[i].z, num[2]);
      num[3] = fmaf(w, o[i].w, num[3]);
    }
    m_run = mx;
  }
  // merge the KP parts of each chunk (lanes c, c + CPL, ...)
#pragma unroll
  for (int off = CPL; off < 64; off <<= 1) {
    const float mo = __shfl_xor(m_run, off);
    const float M = fmaxf(m_run, mo);
    const float fa = (m_run == -INFINITY) ? 0.0f : __builtin_amdgcn_exp2f(m_run - M);
    const float fb = (mo == -INFINITY) ? 0.0f : __builtin_amdgcn_exp2f(mo - M);
    den = den * fa + __shfl_xor(den, off) * fb;
#pragma unroll
    for (int e = 0; e < 4; ++e) num[e] = num[e] * fa + __shfl_xor(num[e], off) * fb;
    m_run = M;
  }
  if (k == 0) {
    const float r = den > 0.0f ? 1.0f / den : 0.0f;
    __half2* dst = reinterpret_cast<__half2*>(out + ((size_t)b * Hq + h0 + h) * D + 4 * c);
    dst[0] = __floats2half2_rn(num[0] * r, num[1] * r);
    dst[1] = __floats2half2_rn(num[2] * r, num[3] * r);
  }
}

template <int D, int G, int HPB>
__global__ __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(2))) void decode_kernel(
    const uint8_t* __restrict__ k_codes, const uint32_t* __restrict__ k_meta,
    const uint8_t* __restrict__ v_codes, const uint32_t* __restrict__ v_meta,
    const __half* __restrict__ q, const int32_t* __restrict__ block_tables,
    const int32_t* __restrict__ seq_lens, float* __restrict__ ws, uint32_t* __restrict__ tickets,
    __half* __restrict__ out, int Hq, int Hkv, int P, int NP, int max_pages, int max_splits,
    int n_hchunks, float scale_log2) {
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

  const int kv = blockIdx.y / n_hchunks;
  const int hc = blockIdx.y % n_hchunks;
  const int b = blockIdx.z;
  const int gq = Hq / Hkv;
  const int h0 = kv * gq + hc * HPB;
  const int nh = min(HPB, gq - hc * HPB);
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform (scalar)
  const int split = blockIdx.x;

  const int L = min(seq_lens[b], max_pages * P);
  if (L <= 0) {  // an empty request: all-zero output rows, written by split 0
    if (split == 0)
      for (int i = tid; i < nh * D; i += kThreads)
        out[((size_t)b * Hq + h0) * D + i] = __float2half(0.0f);
    return;
  }
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

  // ---- this wave's rows: the split's rows in page order, g = wave, wave + 4,
  // ... (the four waves read neighbouring rows of one page at a time)
  const int n_split_pages = pe - pb;
  const int split_rows = n_split_pages * rows_per_page;
  const int my_rows = (split_rows > wave) ? (split_rows - wave + kSplitWaves - 1) / kSplitWaves : 0;
  const size_t head_codes = (size_t)P * (D / 2);
  const size_t page_codes = (size_t)Hkv * head_codes;
  uint8_t* ring = smem[wave][0];
  const uint32_t ring_lds = (uint32_t)(uintptr_t)ring;

  // The split's page IDs, 64 per vector register (lane k holds page pb + k of
  // the group), read with v_readlane when the issue cursor enters a page.
  auto load_group = [&](int grp) {
    const int k = 64 * grp + lane;
    return (k < n_split_pages) ? block_tables[(size_t)b * max_pages + pb + k] : -1;
  };
  int pg_grp = load_group(0);
  int cur_grp = 0;

  // query words of the lane's 32 dims for each head (loaded with the page
  // IDs, unpacked once the first rows' loads are in flight)
  // Slot k of lane j holds head j ^ k when lane j owns head j's softmax
  // (then the reduce-scatter of the unit needs no selects), else head k.
  uint4 qraw[HPB][4];
#pragma unroll
  for (int h = 0; h < HPB; ++h) {
    const int head = h0 + min(kLaneHeads ? (j ^ h) : h, nh - 1);
    const uint4* src = reinterpret_cast<const uint4*>(q + ((size_t)b * Hq + head) * D + 32 * j);
#pragma unroll
    for (int m = 0; m < 4; ++m) qraw[h][m] = src[m];
  }

  // Per-lane parts of the load addresses (the row parts are scalar).
  // LDS placement (d = 128): a DMA lane stores 16 bytes at 16 * lane, so the
  // chunk a lane fetches decides the LDS layout.  K: odd units (position
  // pairs) swap their two positions; V: odd units swap the two 16-byte halves
  // of each lane's 32 bytes; meta: odd groups XOR the position with ROWPOS/2.
  // Each read instruction then spreads its 16-lane passes over all 32 banks.
  constexpr bool kSwizzle = (D == 128);
  const uint32_t k_off = 16u * (kSwizzle ? (lane ^ ((lane >> 1) & 4)) : lane);
  const uint32_t v_off = 16u * (kSwizzle ? (lane ^ ((lane >> 3) & 1)) : lane);
  uint32_t meta_off[META_DMAS];  // LDS word w = (group w / ROWPOS, slot w % ROWPOS)
#pragma unroll
  for (int i = 0; i < META_DMAS; ++i) {
    const int w = 64 * i + lane;
    const int wi = (w < META_WORDS) ? w : 0;
    const int grp = wi / ROWPOS;
    const int pos = (wi % ROWPOS) ^ ((grp & 1) * (ROWPOS / 2));
    meta_off[i] = 4u * (uint32_t)(pos * NG + grp);
  }

  // Issue cursor: the next row to load (page ipk of the split, row irr of the
  // page) and the scalar addresses of that row.
  int ipk = wave / rows_per_page, irr = wave % rows_per_page;
  const uint8_t* ik = k_codes;
  const uint8_t* iv = v_codes;
  size_t im = 0;  // byte offset of the row's (scale, bias) words in k_meta / v_meta
  bool iok = false;
  auto enter_page = [&]() {
    if ((ipk >> 6) != cur_grp) {  // more than 64 pages per split: next 64 IDs
      cur_grp = ipk >> 6;
      pg_grp = load_group(cur_grp);
      wait_vm<0>();  // here, so that the common path carries no pending load
    }
    int page = __builtin_amdgcn_readlane(pg_grp, ipk & 63);
    iok = (unsigned)page < (unsigned)NP;
    if (!iok) page = 0;  // never read past the pool; the positions are masked
    ik = k_codes + page * page_codes + kv * head_codes + (size_t)irr * ROWPOS * (D / 2);
    iv = v_codes + page * page_codes + kv * head_codes + (size_t)irr * ROWPOS * (D / 2);
    im = ((((size_t)page * Hkv + kv) * P) + (size_t)irr * ROWPOS) * NG * 4;
  };
  bool stage_ok[kStages];
  // Loads of the next row into stage ST; past the wave's last row, loads of
  // one 16-byte run by every lane (same count, negligible traffic) keep the
  // number of loads in flight per row constant.
  auto issue = [&](auto st_c, bool real) {
    constexpr int ST = decltype(st_c)::value;
    uint8_t* st = ring + ST * kStageBytes;
    if (real) {
      dma16(ik + k_off, st);
      dma16(ik + 1024 + k_off, st + 1024);
      dma16(iv + v_off, st + 2048);
      dma16(iv + 1024 + v_off, st + 3072);
      const uint8_t* km8 = reinterpret_cast<const uint8_t*>(k_meta) + im;
      const uint8_t* vm8 = reinterpret_cast<const uint8_t*>(v_meta) + im;
#pragma unroll
      for (int i = 0; i < META_DMAS; ++i) {
        dma4(km8 + meta_off[i], st + kCodeBytes + 256 * i);
        dma4(vm8 + meta_off[i], st + kCodeBytes + kMetaBytes / 2 + 256 * i);
      }
      stage_ok[ST] = iok;
      // advance the cursor by kSplitWaves rows
      irr += kSplitWaves;
      if (irr < rows_per_page) {
        ik += kSplitWaves * ROWPOS * (D / 2);
        iv += kSplitWaves * ROWPOS * (D / 2);
        im += kSplitWaves * ROWPOS * NG * 4;
      } else {
        do {
          irr -= rows_per_page;
          ++ipk;
        } while (irr >= rows_per_page);
        if (ipk < n_split_pages) enter_page();
      }
    } else {
#pragma unroll
      for (int i = 0; i < 4; ++i) dma16(k_codes, st + 1024 * i);
#pragma unroll
      for (int i = 0; i < 2 * META_DMAS; ++i) dma4(k_meta, st + kCodeBytes + 256 * i);
      stage_ok[ST] = false;
    }
  };
  wait_vm<0>();  // page IDs and query words (issued together) have arrived
  if (my_rows > 0) enter_page();
  // All stages are in flight while a row is computed: a row's stage is read
  // into registers first and then refilled with the row kStages ahead.
  if (my_rows > 0) {
    issue(std::integral_constant<int, 0>{}, 0 < my_rows);
    issue(std::integral_constant<int, 1>{}, 1 < my_rows);
    issue(std::integral_constant<int, 2>{}, 2 < my_rows);
    if constexpr (kStages == 4) issue(std::integral_constant<int, 3>{}, 3 < my_rows);
  }

  // ---- query pairs in unpack order: word m (dims 8m..8m+7 of the lane's 32),
  // pair k = (dim 8m+k, dim 8m+k+4); odd k pre-divided by 16
  h2 qp[HPB][4][4];
  float qsum[HPB];
#pragma unroll
  for (int h = 0; h < HPB; ++h) {
    float s = 0.0f;
#pragma unroll
    for (int m = 0; m < 4; ++m) {
      const uint4 u = qraw[h][m];
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
    qsum[h] = kLaneHeads ? s * (1.0f / 16777216.0f) : s * scale_log2;
  }
  // logit (log2 units) = kfold * (scale * raw_dot + bias * qsum * 2^-24) in the
  // lane-heads path; kfold * scale * raw_dot + bias * qsum otherwise
  const float kfold = 16777216.0f * scale_log2;  // 2^24
  // Lane-heads path: query sums over the dims that share a scale group with
  // the lane, for the slots whose scale/bias fold happens after the group's
  // lanes are summed (G = 64: slots 0 and 2 after one step; G = 128: slot 0
  // after two steps).
  if constexpr (kLaneHeads && LPP == 4 && G >= 64) {
    qsum[0] += dpp_f(qsum[1], 0xB1);
    qsum[2] += dpp_f(qsum[3], 0xB1);
    if constexpr (G >= 128) qsum[0] += dpp_f(qsum[2], 0x4E);
  }
  if constexpr (kLaneHeads && LPP == 2 && G >= 64) qsum[0] += dpp_f(qsum[1], 0xB1);

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


  // Compute cursor: the first (logical) position of the row; the split's
  // pages are consecutive logical pages, so row g starts at pb * P + g * ROWPOS.
  int t_row = pb * P + wave * ROWPOS;
  const int t_lane = 2 * unit;  // the lane's position pair within a row
  const int odd_unit = kSwizzle ? (unit & 1) : 0;
  const uint32_t lds_k0 = ring_lds + (2 * unit) * (D / 2) + 16 * j + 64 * odd_unit;
  const uint32_t lds_k1 = ring_lds + (2 * unit + 1) * (D / 2) + 16 * j - 64 * odd_unit;
  const uint32_t lds_m =
      ring_lds + kCodeBytes + (g * ROWPOS + ((2 * unit) ^ ((g & 1) * (ROWPOS / 2)))) * 4;
  const uint32_t lds_v0 = ring_lds + 2048 + unit * D + 32 * j + 16 * odd_unit;
  const uint32_t lds_v1 = ring_lds + 2048 + unit * D + 32 * j + 16 - 16 * odd_unit;
  const h2 ones = {(_Float16)1.0f, (_Float16)1.0f};

  int issued_rows = kStages;  // rows whose loads were issued (incl. past the end)
  auto irr_left_impl = [&]() { return issued_rows++ < my_rows; };
  auto row = [&](auto st_c) {
    constexpr int ST = decltype(st_c)::value;
    // wait until only the kStages - 1 rows after this one are in flight
    wait_vm<DMAS_PER_ROW * (kStages - 1)>();
    const bool pg_ok = stage_ok[ST];
    const bool full = pg_ok && t_row + ROWPOS <= t_end;  // wave-uniform
    bool ok0 = true, ok1 = true;
    if (!full) {
      ok0 = pg_ok && t_row + t_lane < t_end;
      ok1 = pg_ok && t_row + t_lane + 1 < t_end;
    }
    uint4 kw0, kw1, vw0, vw1;
    uint2 km, vm;
    lds_read_row<ST * kStageBytes, kMetaBytes / 2>(lds_k0, lds_k1, lds_m, lds_v0, lds_v1, kw0, kw1,
                                                   km, vm, vw0, vw1);
    // the stage is in registers now (the read waits for its data): refill it
    issue(std::integral_constant<int, ST>{}, irr_left_impl());

    // ---- QK partial dot products over the lane's 32 dims
    float d0[HPB], d1[HPB];
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
            if (m == 0 && k == 0) {
              d0[h] = dot2_first(ca[k], qp[h][m][k]);
              d1[h] = dot2_first(cb[k], qp[h][m][k]);
            } else {
              d0[h] = dot2(ca[k], qp[h][m][k], d0[h]);
              d1[h] = dot2(cb[k], qp[h][m][k], d1[h]);
            }
          }
      }
    }
    float v0[HPB], v1[HPB];
    if constexpr (!kLaneHeads) {
      const float sk0 = lo_f(km.x) * kfold, bk0 = hi_f(km.x);
      const float sk1 = lo_f(km.y) * kfold, bk1 = hi_f(km.y);
#pragma unroll
      for (int h = 0; h < HPB; ++h) {
        v0[h] = fmaf(sk0, d0[h], bk0 * qsum[h]);
        v1[h] = fmaf(sk1, d1[h], bk1 * qsum[h]);
      }
    }
    uint32_t vm0 = vm.x, vm1 = vm.y;
    if (!full) {
      vm0 = ok0 ? vm0 : 0u;
      vm1 = ok1 ? vm1 : 0u;
    }
    const h2 sv = as_h2(__builtin_amdgcn_perm(vm1, vm0, 0x05040100u));  // (s_t0, s_t1)
    const uint32_t bv = __builtin_amdgcn_perm(vm1, vm0, 0x07060302u);    // (b_t0, b_t1)
    h2 W[HPB];
    if constexpr (kLaneHeads) {
      // reduce-scatter over the unit (lane j keeps head j = slot 0), folding
      // each group's scale and bias in once the lanes of that group are summed
      float sm0, sm1;
      if constexpr (LPP == 4) {
        float e0[4], e1[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          e0[k] = d0[k];
          e1[k] = d1[k];
          if constexpr (G == 32) {
            e0[k] = fold_meta(km.x, e0[k], qsum[k]);
            e1[k] = fold_meta(km.y, e1[k], qsum[k]);
          }
        }
        float n00 = e0[0] + dpp_f(e0[1], 0xB1), n02 = e0[2] + dpp_f(e0[3], 0xB1);
        float n10 = e1[0] + dpp_f(e1[1], 0xB1), n12 = e1[2] + dpp_f(e1[3], 0xB1);
        if constexpr (G == 64) {
          n00 = fold_meta(km.x, n00, qsum[0]);
          n02 = fold_meta(km.x, n02, qsum[2]);
          n10 = fold_meta(km.y, n10, qsum[0]);
          n12 = fold_meta(km.y, n12, qsum[2]);
        }
        sm0 = n00 + dpp_f(n02, 0x4E);
        sm1 = n10 + dpp_f(n12, 0x4E);
        if constexpr (G >= 128) {
          sm0 = fold_meta(km.x, sm0, qsum[0]);
          sm1 = fold_meta(km.y, sm1, qsum[0]);
        }
      } else {  // LPP == 2
        float e0[2] = {d0[0], d0[1]}, e1[2] = {d1[0], d1[1]};
        if constexpr (G == 32) {
#pragma unroll
          for (int k = 0; k < 2; ++k) {
            e0[k] = fold_meta(km.x, e0[k], qsum[k]);
            e1[k] = fold_meta(km.y, e1[k], qsum[k]);
          }
        }
        sm0 = e0[0] + dpp_f(e0[1], 0xB1);
        sm1 = e1[0] + dpp_f(e1[1], 0xB1);
        if constexpr (G >= 64) {
          sm0 = fold_meta(km.x, sm0, qsum[0]);
          sm1 = fold_meta(km.y, sm1, qsum[0]);
        }
      }
      sm0 *= kfold;
      sm1 *= kfold;
      if (!full) {
        sm0 = ok0 ? sm0 : -INFINITY;
        sm1 = ok1 ? sm1 : -INFINITY;
      }
      if (__builtin_amdgcn_ballot_w64(fmaxf(sm0, sm1) > thr_mine) != 0) {
        const float mx = xor_max_from(fmaxf(sm0, sm1), LPP);
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
          const float mx = xor_max_from(fmaxf(s0[h], s1[h]), 1);
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
    // advance the compute cursor by kSplitWaves rows (positions stay
    // consecutive across pages of the split)
    t_row += kSplitWaves * ROWPOS;
  };

  for (int r0 = 0; r0 < my_rows; r0 += kStages) {
    row(std::integral_constant<int, 0>{});
    if (r0 + 1 < my_rows) row(std::integral_constant<int, 1>{});
    if (r0 + 2 < my_rows) row(std::integral_constant<int, 2>{});
    if constexpr (kStages == 4) {
      if (r0 + 3 < my_rows) row(std::integral_constant<int, 3>{});
    }
  }
  wait_vm<0>();
  if constexpr (kLaneHeads) {
#pragma unroll
    for (int h = 0; h < HPB; ++h) m_run[h] = bcast_head<LPP>(m_mine, h);
  }

  // ---- merge.  Each wave sums its units (lanes of equal j) within 16-lane
  // rows and writes one partial per row into its own ring, which is idle now;
  // after one barrier the split's threads add the four waves' partials,
  // rescaled to the split's maximum.
  constexpr int kRows = 4;  // 16-lane rows per wave
  constexpr int kWaveFloats = kStages * kStageBytes / 4;
  float* part = reinterpret_cast<float*>(ring);   // [kRows][HPB][D] code-unit sums
  float* part_b = part + kRows * HPB * D;          // [kRows][HPB][LPP] bias sums
  float* part_l = part_b + kRows * HPB * LPP;      // [kRows][HPB]
  float* part_m = part_l + kRows * HPB;            // [HPB]
  static_assert(kRows * HPB * (D + LPP + 1) + HPB <= kWaveFloats, "merge partials fit a ring");
  // lane-derived indices recomputed here (volatile), so that none of them
  // stays live through the row loop
  const int lane_e = lane_id_volatile();
  const int row16 = lane_e >> 4;
  const int je = lane_e & 15;
  const bool writer = je < LPP;  // then je is the lane's j
  // reduce and store four sums at a time (the scheduling barrier keeps the
  // rotations from all being issued ahead of the stores, which would need a
  // second register file's worth of temporaries)
#pragma unroll
  for (int h = 0; h < HPB; ++h) {
    float* dst = part + (row16 * HPB + h) * D + 32 * je;
#pragma unroll
    for (int i = 0; i < 32; i += 4) {
      const float r0 = row_units_sum<LPP>(acc[h][i]), r1 = row_units_sum<LPP>(acc[h][i + 1]);
      const float r2 = row_units_sum<LPP>(acc[h][i + 2]), r3 = row_units_sum<LPP>(acc[h][i + 3]);
      if (writer) *reinterpret_cast<float4*>(dst + i) = make_float4(r0, r1, r2, r3);
      __builtin_amdgcn_sched_barrier(0);
    }
    const float bsum = row_units_sum<LPP>(b_acc[h]);
    if (writer) part_b[(row16 * HPB + h) * LPP + je] = bsum;
  }
  if constexpr (kLaneHeads) {
    const float lsum = row_units_sum<LPP>(l_mine);
    if (writer) part_l[row16 * HPB + je] = lsum;
  } else {
#pragma unroll
    for (int h = 0; h < HPB; ++h) {
      const float lsum = row_units_sum<LPP>(l_acc[h]);
      if (writer && je == 0) part_l[row16 * HPB + h] = lsum;
    }
  }
  if (lane_e == 0) {
#pragma unroll
    for (int h = 0; h < HPB; ++h) part_m[h] = m_run[h];
  }
  __syncthreads();

  {
    const float* base = reinterpret_cast<const float*>(smem[0][0]);
    for (int o = wave * 64 + lane_e; o < nh * D; o += 64 * kSplitWaves) {
      const int h = o / D, dd = o % D, jj = dd / 32;
      // undo the 2^-24 (even dims) or 2^-20 (odd dims of each 4) code factor
      const float cf = (dd & 1) ? 1048576.0f : 16777216.0f;
      float mw[kSplitWaves];
      float M = kMinit;
#pragma unroll
      for (int w = 0; w < kSplitWaves; ++w) {
        mw[w] = base[w * kWaveFloats + kRows * HPB * (D + LPP + 1) + h];
        M = fmaxf(M, mw[w]);
      }
      float num = 0.0f, den = 0.0f;
#pragma unroll
      for (int w = 0; w < kSplitWaves; ++w) {
        const float* pw = base + w * kWaveFloats;
        float a = 0.0f, bs = 0.0f, ls = 0.0f;
#pragma unroll
        for (int rr = 0; rr < kRows; ++rr) {
          a += pw[(rr * HPB + h) * D + dd];
          bs += pw[kRows * HPB * D + (rr * HPB + h) * LPP + jj];
          ls += pw[kRows * HPB * (D + LPP) + rr * HPB + h];
        }
        const float f = __builtin_amdgcn_exp2f(mw[w] - M);
        num = fmaf(f, fmaf(a, cf, bs), num);
        den = fmaf(f, ls, den);
      }
      // agent-scope stores write through to the device-coherent level, so the
      // block that combines (on any XCD) reads them without a cache flush
      float* rec = ws + (((size_t)b * Hq + (h0 + h)) * max_splits + split) * (D + 4);
      __hip_atomic_store(&rec[dd], (den > 0.0f) ? num / den : 0.0f, __ATOMIC_RELAXED,
                         __HIP_MEMORY_SCOPE_AGENT);
      if (dd == 0) {
        __hip_atomic_store(&rec[D], M, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_store(&rec[D + 1], den, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
    }
  }

  // ---- the last split of this (request, KV head, head chunk) to finish
  // combines all of them (log-sum-exp), so no second kernel is needed
  wait_vm<0>();     // this thread's records are stored
  __syncthreads();  // ... and every thread's; the merge buffers are free
  __shared__ uint32_t s_ticket;
  uint32_t* ticket = tickets + ((size_t)b * Hkv + kv) * n_hchunks + hc;
  if (tid == 0)
    s_ticket = __hip_atomic_fetch_add(ticket, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  __syncthreads();
  if (s_ticket != (uint32_t)(S - 1)) return;
  if (tid == 0) __hip_atomic_store(ticket, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  combine_splits<D>(ws, out, b, Hq, h0, nh, max_splits, S);

}

template <int D, int G, int HPB>
hipError_t launch_t(const jf_kv_layout& L, const jf_kv_pool_ptrs& pool, const void* q,
                    int32_t B, int32_t Hq, const int32_t* bt, int32_t max_pages,
                    const int32_t* lens, float scale, int32_t max_splits, void* ws, void* out,
                    hipStream_t stream) {
  const int gq = Hq / L.num_kv_heads;
  const int n_hchunks = (gq + HPB - 1) / HPB;
  dim3 grid(max_splits, L.num_kv_heads * n_hchunks, B);
  // completion counters first, then the split records
  uint32_t* tickets = static_cast<uint32_t*>(ws);
  float* records = reinterpret_cast<float*>(static_cast<uint8_t*>(ws) + jfkv::kDecodeCounterBytes);
  hipLaunchKernelGGL((decode_kernel<D, G, HPB>), grid, dim3(kThreads), 0, stream,
                     static_cast<const uint8_t*>(pool.k_codes),
                     static_cast<const uint32_t*>(pool.k_meta),
                     static_cast<const uint8_t*>(pool.v_codes),
                     static_cast<const uint32_t*>(pool.v_meta), static_cast<const __half*>(q),
                     bt, lens, records, tickets, static_cast<__half*>(out), Hq,
                     L.num_kv_heads, L.page_size, L.num_pages, max_pages, max_splits, n_hchunks,
                     scale * kLog2e);
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
