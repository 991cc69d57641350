// Split-K single-query decode attention over the paged 4-bit KV cache
// (gfx950, VALU; no matrix cores: one query row per head is not a dense
// contraction).
//
// The decode kernel reads the compressed pages where they are used instead of
// expanding the cache (Sec. 3.1, "Decode and prefill need different
// kernels"); heads are independent and query heads share their KV head
// (eq. groupattention).  Work is split over page-aligned ranges of each
// request ("split-K"); every split writes an fp32 partial (o, m, l) and a
// second kernel merges them with a log-sum-exp combine, so the workspace is
// bounded by the split cap rather than by the context length.
//
// Mapping (d = 128): a "unit" of D/32 lanes owns one pair of adjacent
// positions; lane j of the unit holds dims 32j..32j+31.  A wave covers 2*64/
// (D/32) positions per row (32 at d = 128); the four waves of a block take
// rows round-robin.  Per position pair a lane issues two 16-byte K loads (one
// per position, row-major codes), two 16-byte V loads (position-paired
// codes), and four 4-byte meta loads.
//
// Arithmetic: codes are turned into exact fp16 pairs with a mask-and-or into
// the mantissa of 1024 followed by one packed fp16 subtract/fma, then
// consumed by v_dot2 (two fp16 products, fp32 accumulate):
//   - QK: the pairs are (dim 8m+k, dim 8m+k+4) of one position, against the
//     matching fp16 query pairs; logit = scale_g * (q . c) + bias_g * sum(q)
//     per group, reduced over the unit's lanes;
//   - PV: the V layout pairs positions, so a word yields (position 2s,
//     position 2s+1) for one dim and v_dot2 against (w_2s, w_2s+1), with
//     w = p * scale (fp16), accumulates both positions at once; the bias part
//     is sum(p * bias) per group, added once at the end.
// Online softmax keeps one running maximum per head per wave; it is refreshed
// only when some logit exceeds it by more than 2 (log2 units), which bounds
// p by 4 (fp16-safe for any fp16 scale) and makes rescaling rare.
#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>

#include "jfkv_internal.h"

namespace {

typedef _Float16 h2 __attribute__((ext_vector_type(2)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kTau = 2.0f;  // lazy-rescale margin, log2 units
constexpr int kThreads = 256;
constexpr int kWaves = kThreads / 64;

__device__ __forceinline__ h2 as_h2(uint32_t u) { return __builtin_bit_cast(h2, u); }
__device__ __forceinline__ uint32_t as_u32(h2 v) { return __builtin_bit_cast(uint32_t, v); }
__device__ __forceinline__ float dot2(h2 a, h2 b, float c) {
  return __builtin_amdgcn_fdot2(a, b, c, false);
}
__device__ __forceinline__ float lo_f(uint32_t u) {
  return (float)__builtin_bit_cast(h2, u).x;
}
__device__ __forceinline__ float hi_f(uint32_t u) {
  return (float)__builtin_bit_cast(h2, u).y;
}

// Word of eight 4-bit codes (nibble n at bits 4n) -> four exact fp16 pairs:
// out[k] = (code of nibble k, code of nibble k+4), k = 0..3.
__device__ __forceinline__ void unpack8(uint32_t w, h2 out[4]) {
  const uint32_t M = 0x64006400u;  // fp16 1024: mantissa ulp 1
  const uint32_t w8 = w >> 8;
  const h2 c1024 = {(_Float16)1024.0f, (_Float16)1024.0f};
  const h2 c64 = {(_Float16)64.0f, (_Float16)64.0f};
  const h2 c16th = {(_Float16)0.0625f, (_Float16)0.0625f};
  out[0] = as_h2((w & 0x000F000Fu) | M) - c1024;                              // 1024 + c
  out[1] = __builtin_elementwise_fma(as_h2((w & 0x00F000F0u) | M), c16th, -c64);  // 1024 + 16c
  out[2] = as_h2((w8 & 0x000F000Fu) | M) - c1024;
  out[3] = __builtin_elementwise_fma(as_h2((w8 & 0x00F000F0u) | M), c16th, -c64);
}

template <int LPP>
__device__ __forceinline__ float unit_sum(float v) {
#pragma unroll
  for (int off = 1; off < LPP; off <<= 1) v += __shfl_xor(v, off);
  return v;
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) v = fmaxf(v, __shfl_xor(v, off));
  return v;
}

// Page-aligned split s of n_pages pages into S parts (remainder first).
__device__ __forceinline__ void split_range(int n_pages, int S, int s, int& pb, int& pe) {
  const int base = n_pages / S, rem = n_pages % S;
  pb = s * base + min(s, rem);
  pe = pb + base + (s < rem ? 1 : 0);
}

template <int D, int HPB>
__global__ __launch_bounds__(kThreads, 2) void decode_split_kernel(
    const uint8_t* __restrict__ k_codes, const uint32_t* __restrict__ k_meta,
    const uint8_t* __restrict__ v_codes, const uint32_t* __restrict__ v_meta,
    const __half* __restrict__ q, const int32_t* __restrict__ block_tables,
    const int32_t* __restrict__ seq_lens, float* __restrict__ ws, int Hq, int Hkv, int P, int G,
    int NP, int max_pages, int max_splits, int n_hchunks, float scale_log2) {
  constexpr int LPP = D / 32;          // lanes per position pair (unit)
  constexpr int UNITS = 64 / LPP;      // units per wave
  constexpr int ROWPOS = 2 * UNITS;    // positions per wave row
  constexpr int NG_MAX = D / 32;       // groups per head at most (G >= 32)
  static_assert(NG_MAX >= 1, "");

  const int split = blockIdx.x;
  const int kv = blockIdx.y / n_hchunks;
  const int hc = blockIdx.y % n_hchunks;
  const int b = blockIdx.z;
  const int gq = Hq / Hkv;
  const int h0 = kv * gq + hc * HPB;
  const int nh = min(HPB, gq - hc * HPB);

  int L = seq_lens[b];
  const int cap = max_pages * P;
  L = min(L, cap);
  if (L <= 0) return;
  const int n_pages = (L + P - 1) / P;
  const int S = min(max_splits, n_pages);
  if (split >= S) return;
  int pb, pe;
  split_range(n_pages, S, split, pb, pe);
  const int t_begin = pb * P;
  const int t_end = min(pe * P, L);

  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int unit = lane / LPP;
  const int j = lane % LPP;
  const int ng = D / G;
  const int g = (32 * j) / G;

  // ---- query pairs in unpack order, per head: word m (dims 8m..8m+7 of the
  // lane's 32), pair k = (dim 8m+k, dim 8m+k+4)
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
      const uint32_t wq[4] = {u.x, u.y, u.z, u.w};  // dims 8m+0..7 as fp16 pairs
      _Float16 e[8];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        e[2 * i] = as_h2(wq[i]).x;
        e[2 * i + 1] = as_h2(wq[i]).y;
      }
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        qp[h][m][k] = h2{e[k], e[k + 4]};
        s += (float)e[k] + (float)e[k + 4];
      }
    }
    qsum[h] = s;
  }

  float m_run[HPB], l_acc[HPB], b_acc[HPB];
  float acc[HPB][32];
#pragma unroll
  for (int h = 0; h < HPB; ++h) {
    m_run[h] = -INFINITY;
    l_acc[h] = 0.0f;
    b_acc[h] = 0.0f;
#pragma unroll
    for (int i = 0; i < 32; ++i) acc[h][i] = 0.0f;
  }

  const size_t head_codes = (size_t)P * (D / 2);
  const size_t page_codes = (size_t)Hkv * head_codes;
  const h2 ones = {(_Float16)1.0f, (_Float16)1.0f};

  for (int row = wave;; row += kWaves) {
    const int t_row = t_begin + row * ROWPOS;
    if (t_row >= t_end) break;
    const int lp = t_row / P;
    const int page = block_tables[(size_t)b * max_pages + lp];
    if ((unsigned)page >= (unsigned)NP) continue;  // never dereferenced
    const int slot0 = (t_row % P) + 2 * unit;
    const int t0 = t_row + 2 * unit;
    const bool ok0 = t0 < t_end, ok1 = t0 + 1 < t_end;

    const size_t ph = (size_t)page * Hkv + kv;
    const uint8_t* kc = k_codes + page * page_codes + kv * head_codes;
    const uint4 kw0 = *reinterpret_cast<const uint4*>(kc + (size_t)slot0 * (D / 2) + 16 * j);
    const uint4 kw1 =
        *reinterpret_cast<const uint4*>(kc + (size_t)(slot0 + 1) * (D / 2) + 16 * j);
    const uint32_t km0 = k_meta[(ph * P + slot0) * ng + g];
    const uint32_t km1 = k_meta[(ph * P + slot0 + 1) * ng + g];
    const uint8_t* vc = v_codes + page * page_codes + kv * head_codes;
    const uint4* vsrc =
        reinterpret_cast<const uint4*>(vc + (size_t)(slot0 >> 1) * D + 32 * j);
    const uint4 vw0 = vsrc[0], vw1 = vsrc[1];
    uint32_t vm0 = v_meta[(ph * P + slot0) * ng + g];
    uint32_t vm1 = v_meta[(ph * P + slot0 + 1) * ng + g];

    // ---- QK partial dot products over the lane's 32 dims
    float d0[HPB], d1[HPB];
#pragma unroll
    for (int h = 0; h < HPB; ++h) d0[h] = d1[h] = 0.0f;
    {
      const uint32_t ka[4] = {kw0.x, kw0.y, kw0.z, kw0.w};
      const uint32_t kb[4] = {kw1.x, kw1.y, kw1.z, kw1.w};
#pragma unroll
      for (int m = 0; m < 4; ++m) {
        h2 ca[4], cb[4];
        unpack8(ka[m], ca);
        unpack8(kb[m], cb);
#pragma unroll
        for (int h = 0; h < HPB; ++h)
#pragma unroll
          for (int k = 0; k < 4; ++k) {
            d0[h] = dot2(ca[k], qp[h][m][k], d0[h]);
            d1[h] = dot2(cb[k], qp[h][m][k], d1[h]);
          }
      }
    }
    const float sk0 = lo_f(km0), bk0 = hi_f(km0), sk1 = lo_f(km1), bk1 = hi_f(km1);
    float s0[HPB], s1[HPB];
    bool need = false;
#pragma unroll
    for (int h = 0; h < HPB; ++h) {
      float a = unit_sum<LPP>(sk0 * d0[h] + bk0 * qsum[h]);
      float c = unit_sum<LPP>(sk1 * d1[h] + bk1 * qsum[h]);
      s0[h] = ok0 ? a * scale_log2 : -INFINITY;
      s1[h] = ok1 ? c * scale_log2 : -INFINITY;
      need |= fmaxf(s0[h], s1[h]) > m_run[h] + kTau;
    }
    if (__builtin_amdgcn_ballot_w64(need) != 0) {
#pragma unroll
      for (int h = 0; h < HPB; ++h) {
        const float mx = wave_max(fmaxf(s0[h], s1[h]));
        if (mx > m_run[h]) {  // wave-uniform
          const float alpha = exp2f(m_run[h] - mx);
          m_run[h] = mx;
          l_acc[h] *= alpha;
          b_acc[h] *= alpha;
#pragma unroll
          for (int i = 0; i < 32; ++i) acc[h][i] *= alpha;
        }
      }
    }
    // ---- PV
    if (!ok0) vm0 = 0u;
    if (!ok1) vm1 = 0u;
    const h2 sv = as_h2(__builtin_amdgcn_perm(vm1, vm0, 0x05040100u));  // (s_t0, s_t1)
    const h2 bv = as_h2(__builtin_amdgcn_perm(vm1, vm0, 0x07060302u));  // (b_t0, b_t1)
    h2 W[HPB];
#pragma unroll
    for (int h = 0; h < HPB; ++h) {
      const float p0 = exp2f(s0[h] - m_run[h]);
      const float p1 = exp2f(s1[h] - m_run[h]);
      const h2 pp = h2{(_Float16)p0, (_Float16)p1};
      l_acc[h] = dot2(pp, ones, l_acc[h]);
      b_acc[h] = dot2(pp, bv, b_acc[h]);
      W[h] = pp * sv;
    }
    const uint32_t va[8] = {vw0.x, vw0.y, vw0.z, vw0.w, vw1.x, vw1.y, vw1.z, vw1.w};
#pragma unroll
    for (int m = 0; m < 8; ++m) {
      h2 c[4];
      unpack8(va[m], c);  // c[k] = (dim 4m+k of t0, dim 4m+k of t1)
#pragma unroll
      for (int h = 0; h < HPB; ++h)
#pragma unroll
        for (int k = 0; k < 4; ++k) acc[h][4 * m + k] = dot2(W[h], c[k], acc[h][4 * m + k]);
    }
  }

  // ---- merge the units of each wave and the waves of the block
  __shared__ float red[kWaves][UNITS][D];
  __shared__ float red_l[kWaves][UNITS];
  __shared__ float red_m[kWaves][HPB];
  if (lane == 0) {
#pragma unroll
    for (int h = 0; h < HPB; ++h) red_m[wave][h] = m_run[h];
  }
  __syncthreads();
#pragma unroll
  for (int h = 0; h < HPB; ++h) {
    float M = -INFINITY;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) M = fmaxf(M, red_m[w][h]);
    const float f = (m_run[h] == -INFINITY) ? 0.0f : exp2f(m_run[h] - M);
#pragma unroll
    for (int i = 0; i < 32; ++i) red[wave][unit][32 * j + i] = (acc[h][i] + b_acc[h]) * f;
    if (j == 0) red_l[wave][unit] = l_acc[h] * f;
    __syncthreads();
    if (threadIdx.x < D && h < nh) {
      float o = 0.0f, l = 0.0f;
      for (int w = 0; w < kWaves; ++w)
        for (int u = 0; u < UNITS; ++u) {
          o += red[w][u][threadIdx.x];
          l += red_l[w][u];
        }
      float* rec = ws + (((size_t)b * Hq + (h0 + h)) * max_splits + split) * (D + 2);
      rec[threadIdx.x] = (l > 0.0f) ? o / l : 0.0f;
      if (threadIdx.x == 0) {
        rec[D] = M;
        rec[D + 1] = l;
      }
    }
    __syncthreads();
  }
}

template <int D>
__global__ __launch_bounds__(D) void decode_combine_kernel(
    const float* __restrict__ ws, const int32_t* __restrict__ seq_lens, __half* __restrict__ out,
    int Hq, int P, int max_pages, int max_splits) {
  const int h = blockIdx.x, b = blockIdx.y, i = threadIdx.x;
  int L = min(seq_lens[b], max_pages * P);
  __half* dst = out + ((size_t)b * Hq + h) * D;
  if (L <= 0) {
    dst[i] = __float2half(0.0f);
    return;
  }
  const int n_pages = (L + P - 1) / P;
  const int S = min(max_splits, n_pages);
  const float* recs = ws + ((size_t)b * Hq + h) * max_splits * (D + 2);
  float M = -INFINITY;
  for (int s = 0; s < S; ++s) M = fmaxf(M, recs[(size_t)s * (D + 2) + D]);
  float num = 0.0f, den = 0.0f;
  if (M != -INFINITY) {
    for (int s = 0; s < S; ++s) {
      const float* r = recs + (size_t)s * (D + 2);
      const float m = r[D];
      if (m == -INFINITY) continue;
      const float w = r[D + 1] * exp2f(m - M);
      num += w * r[i];
      den += w;
    }
  }
  dst[i] = __float2half_rn(den > 0.0f ? num / den : 0.0f);
}

template <int D, int HPB>
hipError_t launch_decode_t(const jf_kv_layout& L, const jf_kv_pool_ptrs& pool, const void* q,
                           int32_t B, int32_t Hq, const int32_t* bt, int32_t max_pages,
                           const int32_t* lens, float scale, int32_t max_splits, void* ws,
                           void* out, hipStream_t stream) {
  const int gq = Hq / L.num_kv_heads;
  const int n_hchunks = (gq + HPB - 1) / HPB;
  dim3 grid(max_splits, L.num_kv_heads * n_hchunks, B);
  hipLaunchKernelGGL((decode_split_kernel<D, HPB>), grid, dim3(kThreads), 0, stream,
                     static_cast<const uint8_t*>(pool.k_codes),
                     static_cast<const uint32_t*>(pool.k_meta),
                     static_cast<const uint8_t*>(pool.v_codes),
                     static_cast<const uint32_t*>(pool.v_meta), static_cast<const __half*>(q),
                     bt, lens, static_cast<float*>(ws), Hq, L.num_kv_heads, L.page_size,
                     L.group_size, L.num_pages, max_pages, max_splits, n_hchunks,
                     scale * kLog2e);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((decode_combine_kernel<D>), dim3(Hq, B), dim3(D), 0, stream,
                     static_cast<const float*>(ws), lens, static_cast<__half*>(out), Hq,
                     L.page_size, max_pages, max_splits);
  return hipGetLastError();
}

template <int D>
hipError_t dispatch_hpb(const jf_kv_layout& L, const jf_kv_pool_ptrs& pool, const void* q,
                        int32_t B, int32_t Hq, const int32_t* bt, int32_t max_pages,
                        const int32_t* lens, float scale, int32_t max_splits, void* ws,
                        void* out, hipStream_t stream) {
  const int gq = Hq / L.num_kv_heads;
  if (gq == 1)
    return launch_decode_t<D, 1>(L, pool, q, B, Hq, bt, max_pages, lens, scale, max_splits, ws,
                                 out, stream);
  if (gq == 2)
    return launch_decode_t<D, 2>(L, pool, q, B, Hq, bt, max_pages, lens, scale, max_splits, ws,
                                 out, stream);
  if (gq % 3 == 0 && gq % 4 != 0)
    return launch_decode_t<D, 3>(L, pool, q, B, Hq, bt, max_pages, lens, scale, max_splits, ws,
                                 out, stream);
  return launch_decode_t<D, 4>(L, pool, q, B, Hq, bt, max_pages, lens, scale, max_splits, ws,
                               out, stream);
}

}  // namespace

namespace jfkv {

hipError_t launch_decode(const jf_kv_layout& L, const jf_kv_pool_ptrs& pool, const void* q,
                         int32_t B, int32_t Hq, const int32_t* bt, int32_t max_pages,
                         const int32_t* lens, float scale, int32_t max_splits, void* ws,
                         void* out, hipStream_t stream) {
  switch (L.head_dim) {
    case 64:
      return dispatch_hpb<64>(L, pool, q, B, Hq, bt, max_pages, lens, scale, max_splits, ws,
                              out, stream);
    case 128:
      return dispatch_hpb<128>(L, pool, q, B, Hq, bt, max_pages, lens, scale, max_splits, ws,
                               out, stream);
    case 256:
      return dispatch_hpb<256>(L, pool, q, B, Hq, bt, max_pages, lens, scale, max_splits, ws,
                               out, stream);
    default:
      return hipErrorInvalidValue;
  }
}

}  // namespace jfkv
