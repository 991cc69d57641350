// Chunked-prefill attention over the paged 4-bit prefix plus the chunk's own
// fp16 rows, on gfx950 bf16 matrix cores (v_mfma_f32_16x16x32_bf16, fp32
// accumulate).
//
// The paper's prefill consumes the compressed history as floating operands
// for a fused attention (Sec. 3.1, "Decode and prefill need different
// kernels", and Appendix A, Table codec: fused page lookup, unpack and
// reconstruction, writing only the operands); eq. layerbytes gives the size
// of the reconstructed operands it bounds by processing head groups
// (eq. groupattention).  Here the reconstruction never leaves the chip: each
// block dequantizes one 64-key tile of K and V at a time into LDS (bf16) and
// consumes it at once, so no reconstructed K/V reaches HBM.
//
// Block = 4 waves, 128 query rows; a row is (chunk position i, query head h of
// the block's KV head), rows ordered position-major.  Each wave owns 32 rows
// (two 16-row MFMA tiles).  Per key tile:
//   S^T = K Q^T   (A = K tile from LDS [key][dim], B = Q^T in registers)
//   online softmax per query row (a lane holds one row of S^T per tile, so
//   row max/sum need only the 4 lanes sharing lane%16)
//   O^T += V^T P^T (A = V^T tile from LDS [dim][key], B = P^T from the S^T
//   accumulators of the same lanes)
// Accumulator layout used (16x16 MFMA): lane l, element r holds row
// 4*(l/16)+r, column l%16.  The k-slots of an operand are whatever the
// hardware pairs between A and B; both sides are filled with the same key
// (or dim) order, so only that output layout matters.
#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>

#include "jfkv_internal.h"

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef _Float16 h2 __attribute__((ext_vector_type(2)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr int kThreads = 256;
constexpr int kRows = 128;      // query rows per block
constexpr int kKeys = 64;       // keys per tile
constexpr int kKPad = 8;        // bf16 padding of a K-tile row
constexpr int kVPad = 8;        // bf16 padding of a V^T-tile row

// Position of key k (0..63) inside a V^T row: within each 32-key block the
// keys 4q..4q+3 and 16+4q..16+4q+3 sit together, so the eight keys one lane
// feeds to a 32-key MFMA step are contiguous.
__device__ __forceinline__ int vperm(int k) {
  const int kk = k & 31;
  return (k & 32) + 8 * ((kk & 15) >> 2) + 4 * (kk >> 4) + (kk & 3);
}

__device__ __forceinline__ float h2f_lo(uint32_t u) { return (float)__builtin_bit_cast(h2, u).x; }
__device__ __forceinline__ float h2f_hi(uint32_t u) { return (float)__builtin_bit_cast(h2, u).y; }

template <int D>
__global__ __launch_bounds__(kThreads) void prefill_kernel(
    const uint8_t* __restrict__ k_codes, const uint32_t* __restrict__ k_meta,
    const uint8_t* __restrict__ v_codes, const uint32_t* __restrict__ v_meta,
    const __half* __restrict__ q, const __half* __restrict__ k_chunk,
    const __half* __restrict__ v_chunk, const int32_t* __restrict__ block_table,
    __half* __restrict__ out, int T, int Hq, int Hkv, int P, int G, int NP, int max_pages,
    int prefix_len, float scale_log2) {
  constexpr int KSTEPS = D / 32;   // MFMA k-steps over head_dim for S^T
  constexpr int DT = D / 16;       // 16-dim tiles of O^T
  __shared__ __attribute__((aligned(16))) __bf16 sK[kKeys][D + kKPad];
  __shared__ __attribute__((aligned(16))) __bf16 sV[D][kKeys + kVPad];

  const int kv = blockIdx.y;
  const int gq = Hq / Hkv;
  const int r0 = blockIdx.x * kRows;
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int l16 = lane & 15, q4 = lane >> 4;

  // ---- Q^T operands: rows of this wave: r0 + 32*wave + 16*n + l16
  bf16x8 qb[2][KSTEPS];
  int row_pos[2];
#pragma unroll
  for (int n = 0; n < 2; ++n) {
    const int r = r0 + 32 * wave + 16 * n + l16;
    const int i = r / gq, hh = r % gq;
    row_pos[n] = (i < T) ? i : -1;
#pragma unroll
    for (int s = 0; s < KSTEPS; ++s) {
      bf16x8 v;
      if (i < T) {
        const uint4 u = *reinterpret_cast<const uint4*>(
            q + ((size_t)i * Hq + kv * gq + hh) * D + 32 * s + 8 * q4);
        const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          v[2 * e] = (__bf16)h2f_lo(w[e]);
          v[2 * e + 1] = (__bf16)h2f_hi(w[e]);
        }
      } else {
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] = (__bf16)0.0f;
      }
      qb[n][s] = v;
    }
  }

  f32x4 acc_o[DT][2];
#pragma unroll
  for (int t = 0; t < DT; ++t)
#pragma unroll
    for (int n = 0; n < 2; ++n) acc_o[t][n] = f32x4{0, 0, 0, 0};
  float m_row[2] = {-INFINITY, -INFINITY}, l_row[2] = {0.0f, 0.0f};

  // last chunk row of this block (causal horizon of its keys)
  const int last_i = min(T - 1, (r0 + kRows - 1) / gq);
  const int n_pre_tiles = (prefix_len + kKeys - 1) / kKeys;
  const int n_chunk_tiles = (last_i + 1 + kKeys - 1) / kKeys;
  const int ng = D / G;
  const size_t head_codes = (size_t)P * (D / 2);
  const size_t page_codes = (size_t)Hkv * head_codes;

  for (int tile = 0; tile < n_pre_tiles + n_chunk_tiles; ++tile) {
    const bool is_pre = tile < n_pre_tiles;
    const int key0 = is_pre ? tile * kKeys : (tile - n_pre_tiles) * kKeys;  // first key
    const int key_lim = is_pre ? prefix_len : T;                           // valid keys < lim
    // ---- stage K (row-major) and V^T (permuted keys) into LDS as bf16
    {
      for (int task = tid; task < kKeys * (D / 32); task += kThreads) {
        const int key = task / (D / 32), c = task % (D / 32);  // 32 dims per task
        const int kk = key0 + key;
        float x[32];
        if (kk < key_lim) {
          if (is_pre) {
            const int page = block_table[kk / P];
            const int slot = kk % P;
            if ((unsigned)page < (unsigned)NP) {
              const size_t ph = (size_t)page * Hkv + kv;
              const uint4 u = *reinterpret_cast<const uint4*>(
                  k_codes + page * page_codes + kv * head_codes + (size_t)slot * (D / 2) + 16 * c);
              const uint32_t m = k_meta[(ph * P + slot) * ng + (32 * c) / G];
              const float sc = h2f_lo(m), bi = h2f_hi(m);
              const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
              for (int e = 0; e < 32; ++e)
                x[e] = fmaf(sc, (float)((w[e >> 3] >> (4 * (e & 7))) & 15u), bi);
            } else {
#pragma unroll
              for (int e = 0; e < 32; ++e) x[e] = 0.0f;
            }
          } else {
            const uint4* src = reinterpret_cast<const uint4*>(
                k_chunk + ((size_t)kk * Hkv + kv) * D + 32 * c);
#pragma unroll
            for (int v4 = 0; v4 < 4; ++v4) {
              const uint4 u = src[v4];
              const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
              for (int e = 0; e < 4; ++e) {
                x[8 * v4 + 2 * e] = h2f_lo(w[e]);
                x[8 * v4 + 2 * e + 1] = h2f_hi(w[e]);
              }
            }
          }
        } else {
#pragma unroll
          for (int e = 0; e < 32; ++e) x[e] = 0.0f;
        }
#pragma unroll
        for (int v8 = 0; v8 < 4; ++v8) {
          bf16x8 b;
#pragma unroll
          for (int e = 0; e < 8; ++e) b[e] = (__bf16)x[8 * v8 + e];
          *reinterpret_cast<bf16x8*>(&sK[key][32 * c + 8 * v8]) = b;
        }
      }
    }
    {
      // V: a thread takes one key pair and 16 dims (D/16 threads per pair)
      for (int task = tid; task < (kKeys / 2) * (D / 16); task += kThreads) {
        const int pair = task / (D / 16), c16 = task % (D / 16);
        const int ka = key0 + 2 * pair;
        float xa[16], xb[16];
        const bool oka = ka < key_lim, okb = ka + 1 < key_lim;
        if (is_pre && oka) {
          const int page = block_table[ka / P];
          const int slot = ka % P;  // even; slot+1 is on the same page
          if ((unsigned)page < (unsigned)NP) {
            const size_t ph = (size_t)page * Hkv + kv;
            const uint4 u = *reinterpret_cast<const uint4*>(
                v_codes + page * page_codes + kv * head_codes + (size_t)(slot >> 1) * D +
                16 * c16);
            const int g = (16 * c16) / G;
            const uint32_t ma = v_meta[(ph * P + slot) * ng + g];
            const uint32_t mb = okb ? v_meta[(ph * P + slot + 1) * ng + g] : 0u;
            const float sa = h2f_lo(ma), ba = h2f_hi(ma), sb = h2f_lo(mb), bb = h2f_hi(mb);
            const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
            for (int uu = 0; uu < 4; ++uu)
#pragma unroll
              for (int e = 0; e < 4; ++e) {
                xa[4 * uu + e] = fmaf(sa, (float)((w[uu] >> (4 * e)) & 15u), ba);
                xb[4 * uu + e] = okb ? fmaf(sb, (float)((w[uu] >> (16 + 4 * e)) & 15u), bb) : 0.0f;
              }
          } else {
#pragma unroll
            for (int e = 0; e < 16; ++e) xa[e] = xb[e] = 0.0f;
          }
        } else if (!is_pre && oka) {
          const uint4* sa = reinterpret_cast<const uint4*>(
              v_chunk + ((size_t)ka * Hkv + kv) * D + 16 * c16);
#pragma unroll
          for (int v4 = 0; v4 < 2; ++v4) {
            const uint4 u = sa[v4];
            const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              xa[8 * v4 + 2 * e] = h2f_lo(w[e]);
              xa[8 * v4 + 2 * e + 1] = h2f_hi(w[e]);
            }
          }
          if (okb) {
            const uint4* sb = reinterpret_cast<const uint4*>(
                v_chunk + ((size_t)(ka + 1) * Hkv + kv) * D + 16 * c16);
#pragma unroll
            for (int v4 = 0; v4 < 2; ++v4) {
              const uint4 u = sb[v4];
              const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
              for (int e = 0; e < 4; ++e) {
                xb[8 * v4 + 2 * e] = h2f_lo(w[e]);
                xb[8 * v4 + 2 * e + 1] = h2f_hi(w[e]);
              }
            }
          } else {
#pragma unroll
            for (int e = 0; e < 16; ++e) xb[e] = 0.0f;
          }
        } else {
#pragma unroll
          for (int e = 0; e < 16; ++e) xa[e] = xb[e] = 0.0f;
        }
        const int col = vperm(2 * pair);  // keys 2p and 2p+1 are adjacent
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          bf16x2 pr = {(__bf16)xa[e], (__bf16)xb[e]};
          *reinterpret_cast<bf16x2*>(&sV[16 * c16 + e][col]) = pr;
        }
      }
    }
    __syncthreads();

    // ---- S^T = K Q^T : 4 key tiles x 2 row tiles
    f32x4 sacc[4][2];
#pragma unroll
    for (int mt = 0; mt < 4; ++mt)
#pragma unroll
      for (int n = 0; n < 2; ++n) {
        f32x4 c = {0, 0, 0, 0};
#pragma unroll
        for (int s = 0; s < KSTEPS; ++s) {
          const bf16x8 a = *reinterpret_cast<const bf16x8*>(&sK[16 * mt + l16][32 * s + 8 * q4]);
          c = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, qb[n][s], c, 0, 0, 0);
        }
        sacc[mt][n] = c;
      }

    // ---- mask, online softmax per row (row = lane's l16 within tile n)
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
          const float p = exp2f(sacc[mt][n][r] - m_use);
          sacc[mt][n][r] = p;
          ls += p;
        }
      ls += __shfl_xor(ls, 16);
      ls += __shfl_xor(ls, 32);
      l_row[n] = l_row[n] * alpha + ls;
#pragma unroll
      for (int t = 0; t < DT; ++t) acc_o[t][n] *= alpha;
    }

    // ---- O^T += V^T P^T : two 32-key steps
#pragma unroll
    for (int s = 0; s < 2; ++s) {
      bf16x8 pb[2];
#pragma unroll
      for (int n = 0; n < 2; ++n)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          pb[n][r] = (__bf16)sacc[2 * s][n][r];
          pb[n][4 + r] = (__bf16)sacc[2 * s + 1][n][r];
        }
#pragma unroll
      for (int t = 0; t < DT; ++t) {
        const bf16x8 a = *reinterpret_cast<const bf16x8*>(&sV[16 * t + l16][32 * s + 8 * q4]);
#pragma unroll
        for (int n = 0; n < 2; ++n)
          acc_o[t][n] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, pb[n], acc_o[t][n], 0, 0, 0);
      }
    }
    __syncthreads();
  }

  // ---- O = acc / l, written as fp16 (lane holds 4 consecutive dims per tile)
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
      __half2 a = __floats2half2_rn(acc_o[t][n][0] * inv, acc_o[t][n][1] * inv);
      __half2 b = __floats2half2_rn(acc_o[t][n][2] * inv, acc_o[t][n][3] * inv);
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
#define JF_PREFILL_ARGS                                                                         \
  static_cast<const uint8_t*>(pool.k_codes), static_cast<const uint32_t*>(pool.k_meta),        \
      static_cast<const uint8_t*>(pool.v_codes), static_cast<const uint32_t*>(pool.v_meta),    \
      static_cast<const __half*>(q), static_cast<const __half*>(k_chunk),                      \
      static_cast<const __half*>(v_chunk), block_table, static_cast<__half*>(out), T, Hq,      \
      L.num_kv_heads, L.page_size, L.group_size, L.num_pages, max_pages, prefix_len,          \
      softmax_scale * kLog2e
  switch (L.head_dim) {
    case 64:
      hipLaunchKernelGGL(prefill_kernel<64>, grid, dim3(kThreads), 0, stream, JF_PREFILL_ARGS);
      break;
    case 128:
      hipLaunchKernelGGL(prefill_kernel<128>, grid, dim3(kThreads), 0, stream, JF_PREFILL_ARGS);
      break;
    case 256:
      hipLaunchKernelGGL(prefill_kernel<256>, grid, dim3(kThreads), 0, stream, JF_PREFILL_ARGS);
      break;
    default:
      return hipErrorInvalidValue;
  }
#undef JF_PREFILL_ARGS
  return hipGetLastError();
}

}  // namespace jfkv
