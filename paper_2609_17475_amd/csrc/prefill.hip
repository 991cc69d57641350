// Chunked-prefill attention over the paged 4-bit prefix plus the chunk's own
// fp16 rows, on gfx950 matrix cores (v_mfma_f32_16x16x32_f16, fp32
// accumulate).
//
// The paper's prefill consumes the compressed history as floating operands
// of a fused attention (Sec. 3.1, "Decode and prefill need different
// kernels"; Appendix A, Table codec: page lookup, unpack and reconstruction
// fused, writing only the operands); eq. layerbytes is the size of those
// reconstructed operands, which it bounds by processing head groups
// (eq. groupattention).  Here nothing reconstructed reaches HBM: each block
// stages one 64-key tile of 4-bit codes at a time into LDS and consumes it.
//
// Exactness: the matrix products run on the codes themselves (integers
// 0..15, exact in fp16) against the exact fp16 query, and the affine
// per-group scale and bias are folded in afterwards:
//   q . k^_t = sum_g s_tg (q_g . c_tg) + b_tg * sum(q_g)
//   sum_t p_t v^_t[i] = sum_t (p_t s_tg) c_t[i] + sum_t p_t b_tg   (i in g)
// so the only roundings beyond fp32 accumulation are p_t to fp16 and the
// product p_t * s_tg to fp16 (both 2^-11 relative, unbiased).  Rounding the
// dequantized values themselves to a 16-bit type instead costs up to half an
// ulp of |v^|, which for large-magnitude channels exceeds the tolerance.
// The chunk's own fp16 rows use the same path with scale 1 and bias 0.
//
// Block = 4 waves, 128 query rows; a row is (chunk position i, query head h
// of the block's KV head), position-major.  Each wave owns 32 rows (two
// 16-row MFMA tiles).  Per key tile:
//   S^T = K Q^T (A = codes tile [key][dim] from LDS, B = Q^T in registers),
//   one accumulator per scale group, folded into S^T; the bias term is one
//   more MFMA whose k-slots carry (b_g, b_g) x (hi(sum q_g), lo(sum q_g));
//   online softmax per query row (a lane holds one row of S^T per tile, so
//   row max and sum need only the 4 lanes sharing lane%16);
//   O^T += V^T P'^T (A = codes tile [dim][key] from LDS, B = p*s per group).
// Accumulator layout used (16x16 MFMA): lane l, element r holds row
// 4*(l/16)+r, column l%16.  Operand k-slots are whatever the hardware pairs
// between A and B; both sides are filled in the same order.
#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>

#include "jfkv_internal.h"

namespace {

typedef _Float16 h8 __attribute__((ext_vector_type(8)));
typedef _Float16 h2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr int kThreads = 256;
constexpr int kRows = 128;  // query rows per block
constexpr int kKeys = 64;   // keys per tile
constexpr int kPad = 8;     // fp16 padding of an LDS tile row
constexpr int kMaxGroups = 8;

// Position of key k (0..63) inside a V^T row: within each 32-key block the
// keys 4q..4q+3 and 16+4q..16+4q+3 sit together, so the eight keys one lane
// feeds to a 32-key MFMA step are contiguous.
__device__ __forceinline__ int vperm(int k) {
  const int kk = k & 31;
  return (k & 32) + 8 * ((kk & 15) >> 2) + 4 * (kk >> 4) + (kk & 3);
}

__device__ __forceinline__ h2 as_h2(uint32_t u) { return __builtin_bit_cast(h2, u); }
__device__ __forceinline__ uint32_t as_u32(h2 v) { return __builtin_bit_cast(uint32_t, v); }
__device__ __forceinline__ float lo_f(uint32_t u) { return (float)as_h2(u).x; }
__device__ __forceinline__ float hi_f(uint32_t u) { return (float)as_h2(u).y; }

// Eight 4-bit codes (nibble n at bits 4n) -> fp16 pairs (n0,n4), (n1,n5),
// (n2,n6), (n3,n7), exact.
__device__ __forceinline__ void unpack8(uint32_t w, h2 out[4]) {
  const uint32_t M = 0x64006400u;  // fp16 1024: mantissa ulp 1
  const uint32_t w8 = w >> 8;
  const h2 c1024 = {(_Float16)1024.0f, (_Float16)1024.0f};
  const h2 c64 = {(_Float16)64.0f, (_Float16)64.0f};
  const h2 c16th = {(_Float16)0.0625f, (_Float16)0.0625f};
  out[0] = as_h2((w & 0x000F000Fu) | M) - c1024;
  out[1] = __builtin_elementwise_fma(as_h2((w & 0x00F000F0u) | M), c16th, -c64);
  out[2] = as_h2((w8 & 0x000F000Fu) | M) - c1024;
  out[3] = __builtin_elementwise_fma(as_h2((w8 & 0x00F000F0u) | M), c16th, -c64);
}

// Dims of one 8-dim chunk are stored in K tiles in unpack order.
__device__ __forceinline__ int kperm8(int e) { return (e >> 1) + 4 * (e & 1); }

template <int D, int G>
__global__ __launch_bounds__(kThreads) void prefill_kernel(
    const uint8_t* __restrict__ k_codes, const uint32_t* __restrict__ k_meta,
    const uint8_t* __restrict__ v_codes, const uint32_t* __restrict__ v_meta,
    const __half* __restrict__ q, const __half* __restrict__ k_chunk,
    const __half* __restrict__ v_chunk, const int32_t* __restrict__ block_table,
    __half* __restrict__ out, int T, int Hq, int Hkv, int P, int NP, int max_pages,
    int prefix_len, float scale_log2) {
  constexpr int KSTEPS = D / 32;  // 32-dim MFMA steps over head_dim
  constexpr int DT = D / 16;      // 16-dim tiles of O^T
  constexpr int ng = D / G;       // scale groups per head
  constexpr int steps_per_group = G / 32;
  static_assert(ng <= kMaxGroups, "");
  __shared__ __attribute__((aligned(16))) _Float16 sK[kKeys][D + kPad];
  __shared__ __attribute__((aligned(16))) _Float16 sV[D][kKeys + kPad];
  __shared__ __attribute__((aligned(16))) uint32_t sKm[kMaxGroups][kKeys];  // (scale, bias)
  __shared__ __attribute__((aligned(16))) uint32_t sVm[kMaxGroups][kKeys];

  const int kv = blockIdx.y;
  const int gq = Hq / Hkv;
  const int r0 = blockIdx.x * kRows;
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int l16 = lane & 15, q4 = lane >> 4;

  // ---- Q^T operands (exact fp16, dims in unpack order) and per-group sums
  h8 qb[2][KSTEPS];
  h8 qsum_b[2];  // bias-MFMA operand: slots (2g, 2g+1) = hi, lo of sum q_g
  int row_pos[2];
#pragma unroll
  for (int n = 0; n < 2; ++n) {
    const int r = r0 + 32 * wave + 16 * n + l16;
    const int i = r / gq, hh = r % gq;
    row_pos[n] = (i < T) ? i : -1;
    float gs[ng];
#pragma unroll
    for (int g = 0; g < ng; ++g) gs[g] = 0.0f;
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
        float part = 0.0f;
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          v[e] = e8[kperm8(e)];
          part += (float)e8[e];
        }
        gs[(32 * s) / G] += part;
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] = (_Float16)0.0f;
      }
      qb[n][s] = v;
    }
    // complete the group sums over the 4 lanes of this row
#pragma unroll
    for (int g = 0; g < ng; ++g) {
      gs[g] += __shfl_xor(gs[g], 16);
      gs[g] += __shfl_xor(gs[g], 32);
    }
    h8 b;
#pragma unroll
    for (int e = 0; e < 8; ++e) b[e] = (_Float16)0.0f;
#pragma unroll
    for (int g = 0; g < ng; ++g) {
      if ((g >> 2) == q4) {
        const _Float16 hi = (_Float16)gs[g];
        const _Float16 lo = (_Float16)(gs[g] - (float)hi);
        b[2 * (g & 3)] = hi;
        b[2 * (g & 3) + 1] = lo;
      }
    }
    qsum_b[n] = b;
  }

  f32x4 acc_o[DT][2];
#pragma unroll
  for (int t = 0; t < DT; ++t)
#pragma unroll
    for (int n = 0; n < 2; ++n) acc_o[t][n] = f32x4{0, 0, 0, 0};
  float m_row[2] = {-INFINITY, -INFINITY}, l_row[2] = {0.0f, 0.0f};
  float bsum[ng][2];
#pragma unroll
  for (int g = 0; g < ng; ++g) bsum[g][0] = bsum[g][1] = 0.0f;

  const int last_i = min(T - 1, (r0 + kRows - 1) / gq);
  const int n_pre_tiles = (prefix_len + kKeys - 1) / kKeys;
  const int n_chunk_tiles = (last_i + 1 + kKeys - 1) / kKeys;
  const size_t head_codes = (size_t)P * (D / 2);
  const size_t page_codes = (size_t)Hkv * head_codes;
  const uint32_t kUnitMeta = 0x00003C00u;  // scale 1.0, bias 0

  for (int tile = 0; tile < n_pre_tiles + n_chunk_tiles; ++tile) {
    const bool is_pre = tile < n_pre_tiles;
    const int key0 = is_pre ? tile * kKeys : (tile - n_pre_tiles) * kKeys;
    const int key_lim = is_pre ? prefix_len : T;

    // ---- stage K codes (or chunk values) [key][dim, unpack order]
    for (int task = tid; task < kKeys * (D / 32); task += kThreads) {
      const int key = task / (D / 32), c = task % (D / 32);
      const int kk = key0 + key;
      h2 x[16];
#pragma unroll
      for (int e = 0; e < 16; ++e) x[e] = h2{(_Float16)0.0f, (_Float16)0.0f};
      if (kk < key_lim) {
        if (is_pre) {
          const int page = block_table[kk / P];
          if ((unsigned)page < (unsigned)NP) {
            const uint4 u = *reinterpret_cast<const uint4*>(
                k_codes + page * page_codes + kv * head_codes + (size_t)(kk % P) * (D / 2) +
                16 * c);
            const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
            for (int m = 0; m < 4; ++m) unpack8(w[m], &x[4 * m]);
          }
        } else {
          const uint4* src =
              reinterpret_cast<const uint4*>(k_chunk + ((size_t)kk * Hkv + kv) * D + 32 * c);
#pragma unroll
          for (int m = 0; m < 4; ++m) {
            const uint4 u = src[m];  // dims 8m..8m+7 as pairs (0,1) (2,3) (4,5) (6,7)
            const h2 a = as_h2(u.x), b = as_h2(u.y), cc = as_h2(u.z), d = as_h2(u.w);
            x[4 * m + 0] = h2{a.x, cc.x};   // (d0, d4)
            x[4 * m + 1] = h2{a.y, cc.y};   // (d1, d5)
            x[4 * m + 2] = h2{b.x, d.x};    // (d2, d6)
            x[4 * m + 3] = h2{b.y, d.y};    // (d3, d7)
          }
        }
      }
#pragma unroll
      for (int m = 0; m < 4; ++m) {
        uint4 v;
        v.x = as_u32(x[4 * m]);
        v.y = as_u32(x[4 * m + 1]);
        v.z = as_u32(x[4 * m + 2]);
        v.w = as_u32(x[4 * m + 3]);
        *reinterpret_cast<uint4*>(&sK[key][32 * c + 8 * m]) = v;
      }
    }
    // ---- stage V codes (or chunk values) transposed [dim][key, permuted]
    for (int task = tid; task < (kKeys / 2) * (D / 16); task += kThreads) {
      const int pair = task / (D / 16), c16 = task % (D / 16);
      const int ka = key0 + 2 * pair;
      const bool oka = ka < key_lim, okb = ka + 1 < key_lim;
      h2 x[16];  // x[e] = (key 2p, key 2p+1) for dim 16*c16 + e
#pragma unroll
      for (int e = 0; e < 16; ++e) x[e] = h2{(_Float16)0.0f, (_Float16)0.0f};
      if (oka) {
        if (is_pre) {
          const int page = block_table[ka / P];
          if ((unsigned)page < (unsigned)NP) {
            const uint4 u = *reinterpret_cast<const uint4*>(
                v_codes + page * page_codes + kv * head_codes + (size_t)((ka % P) >> 1) * D +
                16 * c16);
            const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
            for (int uu = 0; uu < 4; ++uu) unpack8(w[uu], &x[4 * uu]);  // dims 4uu+0..3
            if (!okb) {  // the odd slot is past the prefix: unwritten
#pragma unroll
              for (int e = 0; e < 16; ++e) x[e].y = (_Float16)0.0f;
            }
          }
        } else {
          const uint4* sa =
              reinterpret_cast<const uint4*>(v_chunk + ((size_t)ka * Hkv + kv) * D + 16 * c16);
          const uint4* sb = reinterpret_cast<const uint4*>(
              v_chunk + ((size_t)(ka + 1) * Hkv + kv) * D + 16 * c16);
#pragma unroll
          for (int v4 = 0; v4 < 2; ++v4) {
            const uint4 ua = sa[v4];
            const uint4 ub = okb ? sb[v4] : make_uint4(0, 0, 0, 0);
            const uint32_t wa[4] = {ua.x, ua.y, ua.z, ua.w};
            const uint32_t wb[4] = {ub.x, ub.y, ub.z, ub.w};
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              x[8 * v4 + 2 * e] = h2{as_h2(wa[e]).x, as_h2(wb[e]).x};
              x[8 * v4 + 2 * e + 1] = h2{as_h2(wa[e]).y, as_h2(wb[e]).y};
            }
          }
        }
      }
      const int col = vperm(2 * pair);  // keys 2p and 2p+1 are adjacent
#pragma unroll
      for (int e = 0; e < 16; ++e)
        *reinterpret_cast<uint32_t*>(&sV[16 * c16 + e][col]) = as_u32(x[e]);
    }
    // ---- stage (scale, bias) per key and group; 0 for keys outside the range
    for (int task = tid; task < kKeys * ng; task += kThreads) {
      const int key = task % kKeys, g = task / kKeys;
      const int kk = key0 + key;
      uint32_t km = 0u, vm = 0u;
      if (kk < key_lim) {
        if (is_pre) {
          const int page = block_table[kk / P];
          if ((unsigned)page < (unsigned)NP) {
            const size_t idx = (((size_t)page * Hkv + kv) * P + kk % P) * ng + g;
            km = k_meta[idx];
            vm = v_meta[idx];
          }
        } else {
          km = vm = kUnitMeta;
        }
      }
      sKm[g][key] = km;
      sVm[g][key] = vm;
    }
    __syncthreads();

    // ---- S^T = sum_g s_g (C_g Q_g^T) + bias term; 4 key tiles x 2 row tiles
    f32x4 sacc[4][2];
#pragma unroll
    for (int mt = 0; mt < 4; ++mt) {
      // bias operand: key 16mt + l16, slots (2g, 2g+1) = (b_g, b_g) on lanes q4 == g/4
      h8 kb;
#pragma unroll
      for (int e = 0; e < 8; ++e) kb[e] = (_Float16)0.0f;
#pragma unroll
      for (int g = 0; g < ng; ++g) {
        if ((g >> 2) == q4) {
          const _Float16 bb = as_h2(sKm[g][16 * mt + l16]).y;
          kb[2 * (g & 3)] = bb;
          kb[2 * (g & 3) + 1] = bb;
        }
      }
#pragma unroll
      for (int n = 0; n < 2; ++n)
        sacc[mt][n] = __builtin_amdgcn_mfma_f32_16x16x32_f16(kb, qsum_b[n], f32x4{0, 0, 0, 0}, 0, 0, 0);
#pragma unroll
      for (int g = 0; g < ng; ++g) {
        f32x4 acc[2] = {f32x4{0, 0, 0, 0}, f32x4{0, 0, 0, 0}};
#pragma unroll
        for (int ss = 0; ss < steps_per_group; ++ss) {
          const int s = g * steps_per_group + ss;
          const h8 a = *reinterpret_cast<const h8*>(&sK[16 * mt + l16][32 * s + 8 * q4]);
#pragma unroll
          for (int n = 0; n < 2; ++n)
            acc[n] = __builtin_amdgcn_mfma_f32_16x16x32_f16(a, qb[n][s], acc[n], 0, 0, 0);
        }
        const uint4 mq = *reinterpret_cast<const uint4*>(&sKm[g][16 * mt + 4 * q4]);
        const float sc[4] = {lo_f(mq.x), lo_f(mq.y), lo_f(mq.z), lo_f(mq.w)};
#pragma unroll
        for (int n = 0; n < 2; ++n)
#pragma unroll
          for (int r = 0; r < 4; ++r) sacc[mt][n][r] = fmaf(sc[r], acc[n][r], sacc[mt][n][r]);
      }
    }

    // ---- mask, online softmax per row (row = lane's l16 within tile n)
    _Float16 ph[4][2][4];  // p rounded to fp16, the values the products use
#pragma unroll
    for (int n = 0; n < 2; ++n) {
      const int ip = row_pos[n];
      float mx = -INFINITY;
#pragma unroll
      for (int mt = 0; mt < 4; ++mt)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int kk = key0 + 16 * mt + 4 * q4 + r;
          bool valid = kk < key_lim && ip >= 0;
          if (!is_pre) valid = valid && kk <= ip;
          const float sv = valid ? sacc[mt][n][r] * scale_log2 : -INFINITY;
          sacc[mt][n][r] = sv;
          mx = fmaxf(mx, sv);
        }
      mx = fmaxf(mx, __shfl_xor(mx, 16));
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      const float m_new = fmaxf(m_row[n], mx);
      const float m_use = (m_new == -INFINITY) ? 0.0f : m_new;
      const float alpha = exp2f(m_row[n] - m_use);
      m_row[n] = m_new;
      float ls = 0.0f;
#pragma unroll
      for (int mt = 0; mt < 4; ++mt)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const _Float16 p = (_Float16)exp2f(sacc[mt][n][r] - m_use);
          ph[mt][n][r] = p;
          ls += (float)p;
        }
      ls += __shfl_xor(ls, 16);
      ls += __shfl_xor(ls, 32);
      l_row[n] = l_row[n] * alpha + ls;
#pragma unroll
      for (int t = 0; t < DT; ++t) acc_o[t][n] *= alpha;
#pragma unroll
      for (int g = 0; g < ng; ++g) bsum[g][n] *= alpha;
    }

    // ---- bias sums and scaled P' operands per group; O^T += V^T P'^T
#pragma unroll
    for (int g = 0; g < ng; ++g) {
      uint4 vm4[4];
#pragma unroll
      for (int mt = 0; mt < 4; ++mt)
        vm4[mt] = *reinterpret_cast<const uint4*>(&sVm[g][16 * mt + 4 * q4]);
      h8 pb[2][2];  // [n][s]
#pragma unroll
      for (int n = 0; n < 2; ++n) {
        float bs = 0.0f;
#pragma unroll
        for (int mt = 0; mt < 4; ++mt) {
          const uint32_t mw[4] = {vm4[mt].x, vm4[mt].y, vm4[mt].z, vm4[mt].w};
#pragma unroll
          for (int r = 0; r < 4; ++r) bs = fmaf((float)ph[mt][n][r], hi_f(mw[r]), bs);
          // keys of mt occupy slots (mt&1)*4 .. +3 of step mt>>1
          const h2 s01 = as_h2(__builtin_amdgcn_perm(mw[1], mw[0], 0x05040100u));
          const h2 s23 = as_h2(__builtin_amdgcn_perm(mw[3], mw[2], 0x05040100u));
          const h2 p01 = h2{ph[mt][n][0], ph[mt][n][1]} * s01;
          const h2 p23 = h2{ph[mt][n][2], ph[mt][n][3]} * s23;
          pb[n][mt >> 1][4 * (mt & 1) + 0] = p01.x;
          pb[n][mt >> 1][4 * (mt & 1) + 1] = p01.y;
          pb[n][mt >> 1][4 * (mt & 1) + 2] = p23.x;
          pb[n][mt >> 1][4 * (mt & 1) + 3] = p23.y;
        }
        bs += __shfl_xor(bs, 16);
        bs += __shfl_xor(bs, 32);
        bsum[g][n] += bs;
      }
      // dim tiles of group g: 16t .. 16t+15 within [g*G, (g+1)*G)
#pragma unroll
      for (int t = 0; t < DT; ++t) {
        if ((16 * t) / G != g) continue;
#pragma unroll
        for (int s = 0; s < 2; ++s) {
          const h8 a = *reinterpret_cast<const h8*>(&sV[16 * t + l16][32 * s + 8 * q4]);
#pragma unroll
          for (int n = 0; n < 2; ++n)
            acc_o[t][n] = __builtin_amdgcn_mfma_f32_16x16x32_f16(a, pb[n][s], acc_o[t][n], 0, 0, 0);
        }
      }
    }
    __syncthreads();
  }

  // ---- O = (acc + bias sum of the dim's group) / l, as fp16
#pragma unroll
  for (int n = 0; n < 2; ++n) {
    const int r = r0 + 32 * wave + 16 * n + l16;
    const int i = r / gq, hh = r % gq;
    if (i >= T) continue;
    const float inv = (l_row[n] > 0.0f) ? 1.0f / l_row[n] : 0.0f;
    __half* dst = out + ((size_t)i * Hq + kv * gq + hh) * D;
#pragma unroll
    for (int t = 0; t < DT; ++t) {
      const int d0 = 16 * t + 4 * q4;
      const float bg = bsum[(16 * t) / G][n];
      const __half2 a = __floats2half2_rn((acc_o[t][n][0] + bg) * inv, (acc_o[t][n][1] + bg) * inv);
      const __half2 b = __floats2half2_rn((acc_o[t][n][2] + bg) * inv, (acc_o[t][n][3] + bg) * inv);
      *reinterpret_cast<__half2*>(dst + d0) = a;
      *reinterpret_cast<__half2*>(dst + d0 + 2) = b;
    }
  }
}

}  // namespace

namespace jfkv {

hipError_t launch_prefill(const jf_kv_layout& L, const jf_kv_pool_ptrs& pool, const void* q,
                          const void* k_chunk, const void* v_chunk, int32_t T, int32_t Hq,
                          const int32_t* block_table, int32_t max_pages, int32_t prefix_len,
                          float softmax_scale, void* out, hipStream_t stream) {
  const int gq = Hq / L.num_kv_heads;
  const int64_t rows = (int64_t)T * gq;
  dim3 grid((uint32_t)((rows + kRows - 1) / kRows), L.num_kv_heads);
#define JF_PREFILL_CASE(D_, G_)                                                                 \
  if (L.head_dim == D_ && L.group_size == G_) {                                                 \
    hipLaunchKernelGGL((prefill_kernel<D_, G_>), grid, dim3(kThreads), 0, stream,               \
                       static_cast<const uint8_t*>(pool.k_codes),                               \
                       static_cast<const uint32_t*>(pool.k_meta),                               \
                       static_cast<const uint8_t*>(pool.v_codes),                               \
                       static_cast<const uint32_t*>(pool.v_meta), static_cast<const __half*>(q),\
                       static_cast<const __half*>(k_chunk), static_cast<const __half*>(v_chunk),\
                       block_table, static_cast<__half*>(out), T, Hq, L.num_kv_heads,           \
                       L.page_size, L.num_pages, max_pages, prefix_len,                          \
                       softmax_scale * kLog2e);                                                 \
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
