// Chunked-prefill attention over the paged 4-bit prefix plus the chunk's own
// fp16 rows, on gfx950 matrix cores (v_mfma_f32_16x16x32_f16, fp32
// accumulation).
//
// The paper's prefill consumes the compressed history as floating operands
// of a fused attention (Sec. 3.1, "Decode and prefill need different
// kernels"; Appendix A, Table codec: page lookup, unpack and reconstruction
// fused, writing only the operands); eq. layerbytes is the size of those
// reconstructed operands, which it bounds by processing head groups
// (eq. groupattention).  Here the reconstructed operands never reach HBM:
// a block of waves shares one KV head and reconstructs one 64-key tile of
// K and V at a time into LDS, double-buffered, while the previous tile is
// consumed by the matrix cores.
//
// Operands:
//   K: the tile holds the exact codes (a 4-bit code masked into the low
//      nibble of an fp16 half that holds 1024.0 is 1024 + code exactly, so
//      one AND-OR and one packed subtraction give two codes); the scores of
//      each scale group come from their own accumulator and are scaled in
//      fp32 by scale * |softmax scale|, and the bias part is one more
//      product whose k-slots carry (b_g, b_g) x (hi, lo) of |softmax
//      scale| times the query's fp32 group sums, plus (1, 1) x (hi, lo) of
//      minus the row's running maximum, so the product leaves the exponent
//      of the softmax numerator directly.  Rounding the reconstructed keys
//      to fp16 instead would move the scores of large-magnitude channels by
//      up to half an fp16 ulp.
//   V: two tiles hold (scale * code + bias) / 2 as an fp16 high part and an
//      fp16 low part (the value rounded once to fp32 by one mixed FMA of
//      the code taken as an fp16 subnormal, then split), and each value
//      product runs once per tile;
//      together they carry the reconstructed value to ~2^-21 relative, and
//      the halving keeps every group in fp16 range (with the scale rounded
//      up, bias + 15 * scale may exceed the fp16 maximum by up to 15 ulps
//      of the scale).  The output is doubled at the end.
// The chunk's own rows are fp16 already: K with scale 1 and bias 0, V halved
// (exact but for the last bit of a subnormal), with no low part.
//
// Block = 8 waves sharing KV head kv, 32 query rows per wave (16 at d = 256); a row is
// (chunk position i, query head h of kv), position-major.  Per 64-key tile:
//   S^T = K Q^T      (A = K code tile [key][dim] from LDS, B = Q^T in
//                     registers, per scale group; a lane holds one query
//                     column, 4 keys per 16-key tile, so row max and sum
//                     need the 4 lanes sharing lane % 16 only)
//   online softmax   (one running maximum per query row, raised only when a
//                     tile's maximum exceeds it by more than kTau, so
//                     p <= 2^kTau stays well inside fp16 and rescaling of
//                     the accumulators is rare; the bias product subtracts
//                     the maximum, so the common tile needs one maximum
//                     per lane and a ballot, then the exponentials)
//   O^T += V^T P^T   (A = V^ high and low tiles [dim][key] from LDS,
//                     B = p as fp16)
// Accumulator layout (16x16 MFMA): lane l, element r holds row 4*(l/16)+r,
// column l%16.  Operand k-slots are whatever the hardware pairs between A
// and B; both sides are filled in the same order.
#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>

#include "jfkv_internal.h"

namespace {

typedef _Float16 h8 __attribute__((ext_vector_type(8)));
typedef _Float16 h2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr float kLog2e = 1.4426950408889634f;
// Keys per tile (a page holds whole tiles): 64, or 32 at d = 256, where the
// double-buffered K and two V tiles of 64 keys would not fit in LDS.
template <int D>
constexpr int keys_per_tile() { return D > 128 ? 32 : 64; }
constexpr float kTau = 8.0f;       // lazy-rescale margin, log2 units
constexpr float kMinit = -1e30f;   // initial running maximum (finite)
constexpr float kFoldMax = 32768.0f;  // running maxima the bias product subtracts

constexpr int kWaves = 8;          // waves per block: two per SIMD
// 16-row MFMA tiles of query rows per wave (the registers of d = 256 hold one)
template <int D>
constexpr int row_tiles() { return D > 128 ? 1 : 2; }

__device__ __forceinline__ h2 as_h2(uint32_t u) { return __builtin_bit_cast(h2, u); }
__device__ __forceinline__ uint32_t as_u32(h2 v) { return __builtin_bit_cast(uint32_t, v); }

// Position of key k (0..63) inside a V^T row: within each 32-key block the
// keys 4q..4q+3 and 16+4q..16+4q+3 sit together, so the eight keys one lane
// feeds to a 32-key MFMA step are contiguous (and pairs 2s, 2s+1 adjacent).
__device__ __forceinline__ int vperm(int k) {
  const int kk = k & 31;
  return (k & 32) + 8 * ((kk & 15) >> 2) + 4 * (kk >> 4) + (kk & 3);
}
// Dims of one 8-dim chunk are stored in K tiles in this order (the order the
// nibble unpacking produces): slot e holds dim kperm8(e).
__device__ __forceinline__ int kperm8(int e) { return (e >> 1) + 4 * (e & 1); }

// Nibble 0 of each 16-bit half of w (the caller shifts by 4 n for nibble n)
// as exact fp16 codes: masked into the mantissa of 1024.0 (1024 + c), then
// 1024 subtracted.  (The matrix cores take normal operands here: the same
// codes as subnormals, c * 2^-24, made the kernel about 4 % slower.)
__device__ __forceinline__ h2 code2(uint32_t w) {
  return as_h2((w & 0x000F000Fu) | 0x64006400u) - h2{(_Float16)1024.0f, (_Float16)1024.0f};
}
// The nibbles of a code word under a mask, kept in place: a 4-bit code c in
// bits 0..3 of a 16-bit half is the fp16 subnormal c * 2^-24 exactly, and
// in bits 4..7 it is c * 2^-20 (bits 8 and up would reach the exponent).
__device__ __forceinline__ h2 nib_lo(uint32_t w) { return as_h2(w & 0x000F000Fu); }
__device__ __forceinline__ h2 nib_hi(uint32_t w) { return as_h2(w & 0x00F000F0u); }
// (scale * code + bias) / 2 of the two codes in c (subnormal, as above) as
// an fp16 high part plus an fp16 low part: t is the value rounded once to
// fp32 (s2 = scale / 2 times the code's power of two, b2 = bias / 2, both
// exact), the high part t rounded to fp16, the low part the rounding of the
// (exact) difference.
// (The conversions are spelled out: left to the compiler, each half is
// converted back to fp32 and subtracted, three instructions where one mixed
// FMA does.)
__device__ __forceinline__ uint32_t deq2hl(h2 c, float sa, float ba, float sb, float bb,
                                           uint32_t& lo) {
  const float t0 = fmaf((float)c.x, sa, ba);
  const float t1 = fmaf((float)c.y, sb, bb);
  uint32_t hi;
  asm("v_cvt_pk_f16_f32 %0, %1, %2" : "=v"(hi) : "v"(t0), "v"(t1));
  asm("v_fma_mixlo_f16 %0, %1, -1.0, %2 op_sel_hi:[1,0,0]" : "=v"(lo) : "v"(hi), "v"(t0));
  asm("v_fma_mixhi_f16 %0, %1, -1.0, %2 op_sel:[1,0,0] op_sel_hi:[1,0,0]" : "+v"(lo) : "v"(hi), "v"(t1));
  return hi;
}

__device__ __forceinline__ f32x4 mfma(h8 a, h8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
}

template <int D, int G>
__global__ __launch_bounds__(64 * kWaves) void prefill_kernel(
    const uint8_t* __restrict__ k_codes, const uint32_t* __restrict__ k_meta,
    const uint8_t* __restrict__ v_codes, const uint32_t* __restrict__ v_meta,
    const __half* __restrict__ q, const __half* __restrict__ k_chunk,
    const __half* __restrict__ v_chunk, const int32_t* __restrict__ block_table,
    __half* __restrict__ out, int T, int Hq, int Hkv, int P, int NP, int prefix_len,
    float scale_log2) {
  constexpr int NR = row_tiles<D>();
  constexpr int kThreads = 64 * kWaves;
  constexpr int kRowsPerWave = 16 * NR;
  constexpr int kRows = kRowsPerWave * kWaves;
  constexpr int KSTEPS = D / 32;           // 32-dim MFMA steps of a score
  constexpr int DT = D / 16;               // 16-dim tiles of O^T
  constexpr int NG = D / G;                // scale groups per vector
  constexpr int KP = D + 16;               // K^ row pitch (fp16; 32 bytes of padding keep the
                                           // 16-byte reads of 16 rows on distinct banks)
  constexpr int KT = keys_per_tile<D>();   // keys per tile
  constexpr int MT = KT / 16;              // 16-key MFMA tiles per tile
  constexpr int KS = KT / 32;              // 32-key MFMA steps per tile
  constexpr int VP = KT + 16;              // V^T row pitch (fp16; likewise)
  constexpr int QPK = D / 32;              // 16-byte K code chunks per key
  constexpr int CPV = D / 16;              // 16-byte V code chunks per key pair
  constexpr int KCH = KT * QPK;         // K code chunks per tile
  constexpr int VCH = (KT / 2) * CPV;   // V code chunks per tile
  constexpr int NCH = (KCH + VCH + kThreads - 1) / kThreads;
  static_assert(G >= 32, "a K chunk (32 dims) and a V chunk (16 dims) lie in one group");

  __shared__ __attribute__((aligned(16))) _Float16 sK[2][KT][KP];
  // per key and scale group: scale * |softmax scale| (log2 units), fp32
  __shared__ __attribute__((aligned(16))) float sKm[2][NG][KT];
  // the bias product's K operand per key: slots (2g, 2g+1) of lane group
  // g / 4 hold (b_g, b_g) (groups 0..7), slots (0, 1) of lane group 3 hold
  // (1, 1) (the running maximum's slots); the other slots stay zero
  constexpr int NBQ = (NG + 3) / 4;
  static_assert(NBQ < 3, "lane group 3 carries the running maximum");
  __shared__ __attribute__((aligned(16))) uint32_t sKb[2][KT][4][4];
  __shared__ __attribute__((aligned(16))) _Float16 sV[2][D][VP];   // V^ / 2, high part
  __shared__ __attribute__((aligned(16))) _Float16 sVl[2][D][VP];  // low part (prefix tiles)

  // KV head fastest: the blocks of one KV head land on one XCD (round-robin
  // dispatch over the 8 XCDs), so its tiles are shared in that XCD's L2.
  const int kv = blockIdx.x % Hkv;
  const int rb = blockIdx.x / Hkv;
  const int gq = Hq / Hkv;
  const int r0 = rb * kRows;
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int l16 = lane & 15, q4 = lane >> 4;
  const size_t head_codes = (size_t)P * (D / 2);

  // scores are scaled by |scale| (log2 units) in the exponent; a negative
  // scale negates the query instead (exact).  A positive floor keeps masked
  // (-inf) scores at -inf when the scale is 0.
  const float cabs = fmaxf(fabsf(scale_log2), 1e-30f);
  const _Float16 qsgn = scale_log2 < 0.0f ? (_Float16)-1.0f : (_Float16)1.0f;

  // ---- Q^T operands (exact fp16, dims in K^ storage order)
  h8 qb[NR][KSTEPS];
  // bias-product operand: slots (2g, 2g+1) = hi, lo of |scale| * sum q_g;
  // in lane group 3, slots (0, 1) = hi, lo of minus the running maximum
  h8 qsum_b[NR];
  int row_i[NR];
#pragma unroll
  for (int n = 0; n < NR; ++n) {
    const int r = r0 + kRowsPerWave * wave + 16 * n + l16;
    const int i = r / gq, hh = r % gq;
    row_i[n] = i;
    float gsum[NG];
#pragma unroll
    for (int g = 0; g < NG; ++g) gsum[g] = 0.0f;
#pragma unroll
    for (int s = 0; s < KSTEPS; ++s) {
      h8 v;
      if (i < T) {
        const uint4 u = *reinterpret_cast<const uint4*>(
            q + ((size_t)i * Hq + kv * gq + hh) * D + 32 * s + 8 * q4);
        const uint32_t w[4] = {u.x, u.y, u.z, u.w};
        _Float16 e8[8];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          e8[2 * e] = as_h2(w[e]).x;
          e8[2 * e + 1] = as_h2(w[e]).y;
        }
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          v[e] = e8[kperm8(e)] * qsgn;
          gsum[(32 * s) / G] += (float)v[e];
        }
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] = (_Float16)0.0f;
      }
      qb[n][s] = v;
    }
    // complete the group sums over the 4 lanes of this row
#pragma unroll
    for (int g = 0; g < NG; ++g) {
      gsum[g] += __shfl_xor(gsum[g], 16);
      gsum[g] += __shfl_xor(gsum[g], 32);
    }
    h8 bq;
#pragma unroll
    for (int e = 0; e < 8; ++e) bq[e] = (_Float16)0.0f;
#pragma unroll
    for (int g = 0; g < NG; ++g) {
      if ((g >> 2) == q4) {
        const float gs = gsum[g] * cabs;
        const _Float16 hi = (_Float16)gs;
        bq[2 * (g & 3)] = hi;
        bq[2 * (g & 3) + 1] = (_Float16)(gs - (float)hi);
      }
    }
    qsum_b[n] = bq;
  }

  f32x4 acc_o[DT][NR];
  // m_run: the running maximum of |scale| * score; m_off: what the bias
  // product subtracts from the scores (m_run, or 0 before the first score
  // and where m_run is too large for two fp16 halves); folded: m_off =
  // m_run in every row of the wave (wave-uniform)
  float m_run[NR], l_run[NR], m_off[NR];
  bool folded = false;
#pragma unroll
  for (int n = 0; n < NR; ++n) {
    m_run[n] = kMinit;
    m_off[n] = 0.0f;
    l_run[n] = 0.0f;
#pragma unroll
    for (int t = 0; t < DT; ++t) acc_o[t][n] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
  }

  const int i_min = r0 / gq;
  const int i_max = min(T - 1, (r0 + kRows - 1) / gq);
  const int n_pre = (prefix_len + KT - 1) / KT;
  const int n_chk = i_max / KT + 1;
  const int n_tiles = n_pre + n_chk;

  // ---- prefix tiles: codes and (scale, bias) words of tile j, one 16-byte
  // code chunk (and its one or two meta words) per thread and round.  K
  // chunk c: key c / QPK, dims 32 (c % QPK) ..; V chunk (after the K ones):
  // key pair p = cv % 32, dims 16 (cv / 32) .. (pairs vary fastest across
  // lanes, so the transposed LDS stores spread over the banks).
  uint4 pc[NCH];
  uint32_t pm[NCH][2];
  static_assert(NCH == 1 && KCH % 64 == 0, "one chunk per thread; K and V chunks in whole waves");
  auto tile_page = [&](int j) { return block_table[(j * KT) / P]; };
  // the wave's role (K or V chunks) and the thread's byte offsets within a
  // (page, KV head) run, before the tile's slot offset (buffer loads: the
  // run's base and the slot offset stay in scalar registers)
  const bool k_wave = __builtin_amdgcn_readfirstlane(wave) * 64 < KCH;
  int code_off = 0, meta_off = 0;
  if (tid < KCH) {
    const int key = tid / QPK, qd = tid % QPK;
    code_off = key * (D / 2) + 16 * qd;
    meta_off = 4 * (key * NG + (32 * qd) / G);
  } else if (tid < KCH + VCH) {
    const int cv = tid - KCH, pair = cv % (KT / 2), u16 = cv / (KT / 2);
    code_off = pair * D + 16 * u16;
    meta_off = 4 * (2 * pair * NG + (16 * u16) / G);
  }
  constexpr int kRsrcFlags = 0x00020000;
  auto prefetch = [&](int j, int page) {
    if ((unsigned)page >= (unsigned)NP) return;  // the tile is skipped
    const int slot0 = (j * KT) % P;
    const size_t run = (size_t)page * Hkv + kv;
    const uint8_t* cbase = (k_wave ? k_codes : v_codes) + run * head_codes;
    const uint32_t* mbase = (k_wave ? k_meta : v_meta) + run * P * NG;
    const auto rc = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t*>(cbase), (short)0,
                                                      (int)head_codes, kRsrcFlags);
    const auto rm = __builtin_amdgcn_make_buffer_rsrc(const_cast<uint32_t*>(mbase), (short)0,
                                                      4 * P * NG, kRsrcFlags);
    if (tid < KCH + VCH) {
      const u32x4 u = __builtin_amdgcn_raw_buffer_load_b128(rc, code_off, slot0 * (D / 2), 0);
      pc[0] = make_uint4(u.x, u.y, u.z, u.w);
      pm[0][0] = __builtin_amdgcn_raw_buffer_load_b32(rm, meta_off, 4 * slot0 * NG, 0);
      if (!k_wave) pm[0][1] = __builtin_amdgcn_raw_buffer_load_b32(rm, meta_off + 4 * NG, 4 * slot0 * NG, 0);
    }
  };
  // reconstruct the prefetched tile j into buffer b (keys past the prefix:
  // scale and bias 0, so they are exact zeros)
  auto dequant = [&](int j, int page, int b) {
    if ((unsigned)page >= (unsigned)NP) return;
    const int key0 = j * KT;
#pragma unroll
    for (int k = 0; k < NCH; ++k) {
      const int c = tid + k * kThreads;
      const uint32_t w[4] = {pc[k].x, pc[k].y, pc[k].z, pc[k].w};
      if (c < KCH) {
        const int key = c / QPK, qd = c % QPK;
        const bool on = key0 + key < prefix_len;
#pragma unroll
        for (int m = 0; m < 4; ++m) {
          uint4 o;
          o.x = as_u32(code2(w[m]));
          o.y = as_u32(code2(w[m] >> 4));
          o.z = as_u32(code2(w[m] >> 8));
          o.w = as_u32(code2(w[m] >> 12));
          *reinterpret_cast<uint4*>(&sK[b][key][32 * qd + 8 * m]) = o;
        }
        if ((32 * qd) % G == 0) {
          const int g = (32 * qd) / G;
          const uint32_t mw = on ? pm[k][0] : 0u;
          sKm[b][g][key] = (float)as_h2(mw).x * cabs;
          sKb[b][key][g >> 2][g & 3] = __builtin_amdgcn_perm(mw, mw, 0x03020302u);
        }
      } else if (c < KCH + VCH) {
        const int cv = c - KCH, pair = cv % (KT / 2), u16 = cv / (KT / 2);
        const int kk = key0 + 2 * pair;
        const uint32_t ma = (kk < prefix_len) ? pm[k][0] : 0u;
        const uint32_t mb = (kk + 1 < prefix_len) ? pm[k][1] : 0u;
        // scale / 2 times 2^24 (codes of nibbles 0, 2) or 2^20 (nibbles 1,
        // 3), bias / 2: keys a (low halves) and b (high halves)
        const float sa24 = (float)as_h2(ma).x * 8388608.0f, ba = (float)as_h2(ma).y * 0.5f;
        const float sb24 = (float)as_h2(mb).x * 8388608.0f, bb = (float)as_h2(mb).y * 0.5f;
        const float sa20 = sa24 * 0.0625f, sb20 = sb24 * 0.0625f;
        const int col = vperm(2 * pair);
#pragma unroll
        for (int m = 0; m < 4; ++m) {
          const int d0 = 16 * u16 + 4 * m;
          const uint32_t w8 = w[m] >> 8;
          const h2 c4[4] = {nib_lo(w[m]), nib_hi(w[m]), nib_lo(w8), nib_hi(w8)};
#pragma unroll
          for (int n = 0; n < 4; ++n) {
            uint32_t lo;
            const uint32_t hi = (n & 1) ? deq2hl(c4[n], sa20, ba, sb20, bb, lo)
                                        : deq2hl(c4[n], sa24, ba, sb24, bb, lo);
            *reinterpret_cast<uint32_t*>(&sV[b][d0 + n][col]) = hi;
            *reinterpret_cast<uint32_t*>(&sVl[b][d0 + n][col]) = lo;
          }
        }
      }
    }
  };
  // the chunk's own fp16 rows j*64 .. into buffer b (rows past T: zeros)
  auto stage_chunk = [&](int j, int b) {
    const int key0 = j * KT;
#pragma unroll
    for (int k = 0; k < NCH; ++k) {
      const int c = tid + k * kThreads;
      if (c < KCH) {
        const int key = c / QPK, qd = c % QPK;
        const int kk = key0 + key;
        const uint4* src = reinterpret_cast<const uint4*>(k_chunk + ((size_t)kk * Hkv + kv) * D + 32 * qd);
#pragma unroll
        for (int m = 0; m < 4; ++m) {
          const uint4 u = (kk < T) ? src[m] : make_uint4(0, 0, 0, 0);
          // dims (0,1) (2,3) (4,5) (6,7) -> storage order (0,4) (1,5) (2,6) (3,7)
          uint4 o;
          o.x = __builtin_amdgcn_perm(u.z, u.x, 0x05040100u);
          o.y = __builtin_amdgcn_perm(u.z, u.x, 0x07060302u);
          o.z = __builtin_amdgcn_perm(u.w, u.y, 0x05040100u);
          o.w = __builtin_amdgcn_perm(u.w, u.y, 0x07060302u);
          *reinterpret_cast<uint4*>(&sK[b][key][32 * qd + 8 * m]) = o;
        }
        if ((32 * qd) % G == 0) {
          const int g = (32 * qd) / G;
          sKm[b][g][key] = cabs;  // scale 1, bias 0
          sKb[b][key][g >> 2][g & 3] = 0u;
        }
      } else if (c < KCH + VCH) {
        const int cv = c - KCH, pair = cv % (KT / 2), u16 = cv / (KT / 2);
        const int kk = key0 + 2 * pair;
        const uint4* sa = reinterpret_cast<const uint4*>(v_chunk + ((size_t)kk * Hkv + kv) * D + 16 * u16);
        const uint4* sb = reinterpret_cast<const uint4*>(v_chunk + ((size_t)(kk + 1) * Hkv + kv) * D + 16 * u16);
        const int col = vperm(2 * pair);
#pragma unroll
        for (int hv = 0; hv < 2; ++hv) {
          const uint4 ua = (kk < T) ? sa[hv] : make_uint4(0, 0, 0, 0);
          const uint4 ub = (kk + 1 < T) ? sb[hv] : make_uint4(0, 0, 0, 0);
          const uint32_t wa[4] = {ua.x, ua.y, ua.z, ua.w};
          const uint32_t wb[4] = {ub.x, ub.y, ub.z, ub.w};
          const h2 half = {(_Float16)0.5f, (_Float16)0.5f};
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int d0 = 16 * u16 + 8 * hv + 2 * e;
            *reinterpret_cast<uint32_t*>(&sV[b][d0][col]) =
                as_u32(as_h2(__builtin_amdgcn_perm(wb[e], wa[e], 0x05040100u)) * half);
            *reinterpret_cast<uint32_t*>(&sV[b][d0 + 1][col]) =
                as_u32(as_h2(__builtin_amdgcn_perm(wb[e], wa[e], 0x07060302u)) * half);
          }
        }
      }
    }
  };

  // ---- one tile from buffer b: scores, online softmax, value products
  auto compute = [&](int b, int key0, int key_lim, bool chunk_tile) {
    // matrix-core sections at raised wave priority: of the two waves of a
    // SIMD, the one issuing matrix products goes first and the other's
    // vector work fills the cycles between them
    __builtin_amdgcn_s_setprio(1);
    // bias part first (key 16 mt + l16, slots (2g, 2g+1) = (b_g, b_g) on
    // lanes q4 == g / 4), minus the running maximum m_off (lane group 3);
    // it seeds the folded scores
    f32x4 sacc[MT][NR];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
      const h8 kb = *reinterpret_cast<const h8*>(&sKb[b][16 * mt + l16][q4][0]);
#pragma unroll
      for (int n = 0; n < NR; ++n) sacc[mt][n] = mfma(kb, qsum_b[n], f32x4{0.0f, 0.0f, 0.0f, 0.0f});
    }
    // code products per scale group, scaled in fp32 (32-key halves in turn,
    // to bound the live accumulators)
#pragma unroll
    for (int mh = 0; mh < KS; ++mh) {
#pragma unroll
      for (int g = 0; g < NG; ++g) {
        f32x4 acc[2][NR];
#pragma unroll
        for (int x = 0; x < 2; ++x)
#pragma unroll
          for (int n = 0; n < NR; ++n) acc[x][n] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
        for (int ss = 0; ss < G / 32; ++ss) {
          const int s = g * (G / 32) + ss;
#pragma unroll
          for (int x = 0; x < 2; ++x) {
            const h8 a = *reinterpret_cast<const h8*>(&sK[b][16 * (2 * mh + x) + l16][32 * s + 8 * q4]);
#pragma unroll
            for (int n = 0; n < NR; ++n) acc[x][n] = mfma(a, qb[n][s], acc[x][n]);
          }
        }
#pragma unroll
        for (int x = 0; x < 2; ++x) {
          const int mt = 2 * mh + x;
          const float4 sc4 = *reinterpret_cast<const float4*>(&sKm[b][g][16 * mt + 4 * q4]);
          const float sc[4] = {sc4.x, sc4.y, sc4.z, sc4.w};
#pragma unroll
          for (int n = 0; n < NR; ++n)
#pragma unroll
            for (int r = 0; r < 4; ++r) sacc[mt][n][r] = fmaf(sc[r], acc[x][n][r], sacc[mt][n][r]);
        }
      }
    }
    // interleave the matrix products with the folds and LDS reads around
    // them (the scheduler's single-wave MFMA interleaving)
    __builtin_amdgcn_iglp_opt(1);
    __builtin_amdgcn_s_setprio(0);
    // keys past the limit, and (chunk tiles) keys after the row's position
    const bool need_mask = key0 + KT > key_lim || (chunk_tile && key0 + KT - 1 > i_min);
    if (need_mask) {
#pragma unroll
      for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int n = 0; n < NR; ++n)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int kk = key0 + 16 * mt + 4 * q4 + r;
            const bool ok = kk < key_lim && (!chunk_tile || kk <= row_i[n]);
            sacc[mt][n][r] = ok ? sacc[mt][n][r] : -INFINITY;
          }
    }
    // sacc = |scale| * score - m_off.  Fast path: m_off is the running
    // maximum in every row and no score exceeds it by more than kTau, which
    // one maximum per lane and one ballot decide
    float mx = sacc[0][0][0];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
      for (int n = 0; n < NR; ++n)
#pragma unroll
        for (int r = (mt == 0 && n == 0) ? 1 : 0; r < 4; r += 2)
          mx = fmaxf(fmaxf(mx, sacc[mt][n][r]), r + 1 < 4 ? sacc[mt][n][r + 1] : mx);
    // (the slow path works with selects, not per-lane branches: a row whose
    // maximum stays has alpha = 1 and delta = 0; the output accumulators
    // are rescaled after the exponentials, when the scores are no longer
    // live)
    const bool slow = !folded || __builtin_amdgcn_ballot_w64(mx > kTau) != 0;
    float alpha[NR];
    if (slow) {
      bool unfolded = false;
#pragma unroll
      for (int n = 0; n < NR; ++n) {
        float rm = fmaxf(fmaxf(sacc[0][n][0], sacc[0][n][1]), fmaxf(sacc[0][n][2], sacc[0][n][3]));
#pragma unroll
        for (int mt = 1; mt < MT; ++mt)
          rm = fmaxf(rm, fmaxf(fmaxf(sacc[mt][n][0], sacc[mt][n][1]),
                               fmaxf(sacc[mt][n][2], sacc[mt][n][3])));
        rm = fmaxf(rm, __shfl_xor(rm, 16));
        rm = fmaxf(rm, __shfl_xor(rm, 32));
        const float tm = rm + m_off[n];  // the tile's maximum of |scale| * score
        const bool raise = tm > m_run[n] + kTau;
        // a new maximum is rounded to a sum of two fp16 halves, so that the
        // bias product subtracts it exactly
        const _Float16 th = (_Float16)tm;
        const float tr = (float)th + (float)(_Float16)(tm - (float)th);
        const float mnew = fabsf(tm) < kFoldMax ? tr : tm;
        alpha[n] = raise ? __builtin_amdgcn_exp2f(m_run[n] - mnew) : 1.0f;
        m_run[n] = raise ? mnew : m_run[n];
        l_run[n] *= alpha[n];
        // this tile's scores relative to m_run, and the next tiles' m_off
        const bool valid = m_run[n] > kMinit;
        const float delta = valid ? m_run[n] - m_off[n] : 0.0f;
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
#pragma unroll
          for (int r = 0; r < 4; ++r) sacc[mt][n][r] -= delta;
        const bool fold = valid && fabsf(m_run[n]) < kFoldMax;
        m_off[n] = fold ? m_run[n] : 0.0f;
        unfolded = unfolded || !fold;
        const _Float16 oh = (_Float16)m_off[n];
        const _Float16 ol = (_Float16)(m_off[n] - (float)oh);
        qsum_b[n][0] = q4 == 3 ? -oh : qsum_b[n][0];
        qsum_b[n][1] = q4 == 3 ? -ol : qsum_b[n][1];
      }
      folded = __builtin_amdgcn_ballot_w64(unfolded) == 0;
    }
    // p = 2^(s |scale| - m) as fp16; P^T operand of 32-key step k: the
    // lane's keys 4 q4 .. of 16-key tiles 2k and 2k + 1
    h8 pb[NR][KS];
    u32x4 pw[NR][KS];  // the same, as fp16 pairs
    const h2 ones = {(_Float16)1.0f, (_Float16)1.0f};
#pragma unroll
    for (int n = 0; n < NR; ++n) {
#pragma unroll
      for (int mt = 0; mt < MT; ++mt) {
        const float p0 = __builtin_amdgcn_exp2f(sacc[mt][n][0]);
        const float p1 = __builtin_amdgcn_exp2f(sacc[mt][n][1]);
        const float p2 = __builtin_amdgcn_exp2f(sacc[mt][n][2]);
        const float p3 = __builtin_amdgcn_exp2f(sacc[mt][n][3]);
        const h2 a = {(_Float16)p0, (_Float16)p1};
        const h2 c = {(_Float16)p2, (_Float16)p3};
        l_run[n] = __builtin_amdgcn_fdot2(a, ones, l_run[n], false);
        l_run[n] = __builtin_amdgcn_fdot2(c, ones, l_run[n], false);
        pw[n][mt >> 1][2 * (mt & 1) + 0] = as_u32(a);
        pw[n][mt >> 1][2 * (mt & 1) + 1] = as_u32(c);
      }
    }
#pragma unroll
    for (int n = 0; n < NR; ++n)
#pragma unroll
      for (int k = 0; k < KS; ++k) pb[n][k] = __builtin_bit_cast(h8, pw[n][k]);
    if (slow) {
#pragma unroll
      for (int n = 0; n < NR; ++n)
#pragma unroll
        for (int t = 0; t < DT; ++t) acc_o[t][n] *= alpha[n];
    }
    __builtin_amdgcn_s_setprio(1);
#pragma unroll
    for (int t = 0; t < DT; ++t)
#pragma unroll
      for (int k = 0; k < KS; ++k) {
        const h8 a = *reinterpret_cast<const h8*>(&sV[b][16 * t + l16][32 * k + 8 * q4]);
#pragma unroll
        for (int n = 0; n < NR; ++n) acc_o[t][n] = mfma(a, pb[n][k], acc_o[t][n]);
      }
    if (!chunk_tile) {  // the low parts of reconstructed values (block-uniform)
#pragma unroll
      for (int t = 0; t < DT; ++t)
#pragma unroll
        for (int k = 0; k < KS; ++k) {
          const h8 a = *reinterpret_cast<const h8*>(&sVl[b][16 * t + l16][32 * k + 8 * q4]);
#pragma unroll
          for (int n = 0; n < NR; ++n) acc_o[t][n] = mfma(a, pb[n][k], acc_o[t][n]);
        }
    }
    // the same interleaving for the value products, the exponentials and the
    // row sums
    __builtin_amdgcn_iglp_opt(1);
    __builtin_amdgcn_s_setprio(0);
  };

  for (int i = tid; i < 2 * KT * 4 * 4; i += kThreads)
    (&sKb[0][0][0][0])[i] = (i & 15) == 12 ? 0x3C003C00u : 0u;  // (1, 1) in slots (0, 1) of lane group 3
  __syncthreads();

  // ---- tiles 0 .. n_pre - 1 (prefix), then the chunk's; double-buffered:
  // tile j + 1 is reconstructed and tile j + 2's codes are fetched while
  // tile j is computed; one barrier per tile.  Waves w and w + 4 share a
  // SIMD; the first half (the K chunks: the lighter reconstruction) does
  // its part before the tile's products and the second half (the V chunks)
  // after them, so that on each SIMD one wave's vector work meets the
  // other's matrix products (measured 1.5 % faster than the other order).
  int page_pf = -1;     // page of the tile in the prefetch registers
  int page_buf[2] = {0, 0};
  if (n_pre > 0) {
    page_pf = tile_page(0);
    prefetch(0, page_pf);
    dequant(0, page_pf, 0);
    page_buf[0] = page_pf;
    if (n_pre > 1) {
      page_pf = tile_page(1);
      prefetch(1, page_pf);
    }
  } else {
    stage_chunk(0, 0);
  }
  __syncthreads();
  const bool early = wave < kWaves / 2;  // wave-uniform
  for (int j = 0; j < n_tiles; ++j) {
    const int b = j & 1;
    // this thread's part of tile j + 1 into buffer b ^ 1, and tile j + 2's codes
    auto prep = [&]() {
      if (j + 1 < n_tiles) {
        if (j + 1 < n_pre) {
          dequant(j + 1, page_pf, b ^ 1);
          page_buf[b ^ 1] = page_pf;
        } else {
          stage_chunk(j + 1 - n_pre, b ^ 1);
          page_buf[b ^ 1] = 0;
        }
      }
      if (j + 2 < n_pre) {
        page_pf = tile_page(j + 2);
        prefetch(j + 2, page_pf);
      }
    };
    const int page_cur = page_buf[b];
    if (early) prep();
    const bool chunk_tile = j >= n_pre;
    if (chunk_tile)
      compute(b, (j - n_pre) * KT, T, true);
    else if ((unsigned)page_cur < (unsigned)NP)  // a tile on an invalid page is skipped
      compute(b, j * KT, prefix_len, false);
    if (!early) prep();
    __syncthreads();
  }

  // ---- O = acc / l, as fp16
#pragma unroll
  for (int n = 0; n < NR; ++n) {
    const int r = r0 + kRowsPerWave * wave + 16 * n + l16;
    const int i = r / gq, hh = r % gq;
    // the row's sum: the four lanes of a query column hold disjoint keys
    float l = l_run[n] + __shfl_xor(l_run[n], 16);
    l += __shfl_xor(l, 32);
    if (i >= T) continue;
    const float inv = (l > 0.0f) ? 2.0f / l : 0.0f;  // (the value tiles hold V / 2)
    __half* dst = out + ((size_t)i * Hq + kv * gq + hh) * D;
#pragma unroll
    for (int t = 0; t < DT; ++t) {
      const int d0 = 16 * t + 4 * q4;
      const __half2 a = __floats2half2_rn(acc_o[t][n][0] * inv, acc_o[t][n][1] * inv);
      const __half2 c = __floats2half2_rn(acc_o[t][n][2] * inv, acc_o[t][n][3] * inv);
      uint2 v;
      v.x = __builtin_bit_cast(uint32_t, a);
      v.y = __builtin_bit_cast(uint32_t, c);
      *reinterpret_cast<uint2*>(dst + d0) = v;
    }
  }
}

}  // namespace

namespace jfkv {

hipError_t launch_prefill(const jf_kv_layout& L, const jf_kv_pool_ptrs& pool, const void* q,
                          const void* k_chunk, const void* v_chunk, int32_t T, int32_t Hq,
                          const int32_t* block_table, int32_t max_pages, int32_t prefix_len,
                          float softmax_scale, void* out, hipStream_t stream) {
  (void)max_pages;  // validated on the host: prefix_len <= max_pages * page_size
  const int gq = Hq / L.num_kv_heads;
  const int64_t rows = (int64_t)T * gq;
#define JF_PREFILL_CASE(D_, G_)                                                                 \
  if (L.head_dim == D_ && L.group_size == G_) {                                                 \
    constexpr int kRowsB = 16 * row_tiles<D_>() * kWaves;                                      \
    const int64_t n_rb = (rows + kRowsB - 1) / kRowsB;                                          \
    dim3 grid((uint32_t)(n_rb * L.num_kv_heads));                                               \
    hipLaunchKernelGGL((prefill_kernel<D_, G_>), grid, dim3(64 * kWaves), 0, stream,    \
                       static_cast<const uint8_t*>(pool.k_codes),                               \
                       static_cast<const uint32_t*>(pool.k_meta),                               \
                       static_cast<const uint8_t*>(pool.v_codes),                               \
                       static_cast<const uint32_t*>(pool.v_meta), static_cast<const __half*>(q),\
                       static_cast<const __half*>(k_chunk), static_cast<const __half*>(v_chunk),\
                       block_table, static_cast<__half*>(out), T, Hq, L.num_kv_heads,           \
                       L.page_size, L.num_pages, prefix_len, softmax_scale * kLog2e);           \
    return hipGetLastError();                                                                   \
  }
  JF_PREFILL_CASE(64, 32)
  JF_PREFILL_CASE(64, 64)
  JF_PREFILL_CASE(128, 32)
  JF_PREFILL_CASE(128, 64)
  JF_PREFILL_CASE(128, 128)
  JF_PREFILL_CASE(256, 32)
  JF_PREFILL_CASE(256, 64)
  JF_PREFILL_CASE(256, 128)
#undef JF_PREFILL_CASE
  return hipErrorInvalidValue;
}

}  // namespace jfkv
