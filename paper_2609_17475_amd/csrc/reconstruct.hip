// Page -> operand reconstruction for SDPA-style consumers (Background,
// "Stored format is not execution format", eq. layerbytes; Sec. 3.1, "Finish
// one head group before starting the next", eq. groupattention; Appendix A,
// Table codec, reconstruction kernel).  For one request and one group of g
// KV heads, the 4-bit pages of positions 0 .. n - 1 are read through the page
// table and written as contiguous fp16 K and V operands [g][n][d]: 2 g n d 2
// bytes, the only temporary storage a grouped prefill needs.
//
// Each element is the exact value s * q + b rounded once to fp16.  One fp32
// FMA gives s * q + b rounded to fp32 (s * q is exact: an 11-bit scale times
// a 4-bit code); converting that to fp16 rounds a second time, which can
// differ from rounding the exact value only when the fp32 result lies exactly
// on an fp16 rounding midpoint (or in fp16's subnormal range, where the
// midpoint pattern differs).  Those results are detected with two integer
// tests and recomputed exactly: the fp32 sum's error by TwoSum (exact), the
// sum rounded to odd in fp32 (toward zero, last bit set when inexact), then
// to fp16 (rounding to odd with 13 spare bits makes the second rounding
// exact).
//
// Work: a lane reads 8 elements' codes of a position (K) or of a pair of
// positions (V, stored position-paired) and their groups' (scale, bias)
// words, and writes 8 fp16 values (16 bytes) per position, so a wave reads
// consecutive positions' codes as one contiguous run and writes their
// operands contiguously.  Each lane keeps kIters loads in flight.
#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "jfkv.h"
#include "jfkv_internal.h"

namespace {

constexpr int kWaves = 4;
constexpr int kIters = 4;  // loads in flight per lane

// fp16 of s * q + b rounded once, via fp32 rounded to odd (see above).
__device__ __forceinline__ float to_odd(float s, float q, float b) {
  const float a = s * q;  // exact
  const float hi = a + b;
  const float bb = hi - a;
  const float err = (a - (hi - bb)) + (b - bb);  // a + b = hi + err exactly
  uint32_t u = __builtin_bit_cast(uint32_t, hi);
  if (err != 0.0f) {
    if ((err < 0.0f) != (hi < 0.0f)) u -= 1u;  // hi was rounded away from zero
    u |= 1u;
  }
  return __builtin_bit_cast(float, u);
}

// fp32 values whose conversion to fp16 may differ from rounding the exact
// value they approximate: an fp16 rounding midpoint of the normal range (the
// 13 bits below fp16's precision are 1000000000000), or magnitudes below
// 2^-14 (fp16 subnormals).
__device__ __forceinline__ bool near_midpoint(float x) {
  const uint32_t u = __builtin_bit_cast(uint32_t, x);
  return (u & 0x1FFFu) == 0x1000u || (u & 0x7FFFFFFFu) < 0x38800000u;
}

// fp16 of the eight elements of one code word (element k at bits 4k) with
// the group's (scale, bias) word; the exact path for the whole wave when any
// lane's fp32 result may round differently from the exact value.
__device__ __forceinline__ uint4 emit8(uint32_t cw, uint32_t mw) {
  const float s = __half2float(__ushort_as_half((unsigned short)(mw & 0xFFFFu)));
  const float b = __half2float(__ushort_as_half((unsigned short)(mw >> 16)));
  const uint32_t lo = cw & 0x0F0F0F0Fu, hi4 = (cw >> 4) & 0x0F0F0F0Fu;
  float q[8];
#pragma unroll
  for (int k = 0; k < 4; ++k) {
    q[2 * k] = (float)((lo >> (8 * k)) & 0xFFu);       // element 2 k
    q[2 * k + 1] = (float)((hi4 >> (8 * k)) & 0xFFu);  // element 2 k + 1
  }
  float x[8];
  bool risky = false;
#pragma unroll
  for (int k = 0; k < 8; ++k) {
    x[k] = fmaf(s, q[k], b);
    risky |= near_midpoint(x[k]);
  }
  if (__builtin_amdgcn_ballot_w64(risky) != 0) {
#pragma unroll
    for (int k = 0; k < 8; ++k) x[k] = to_odd(s, q[k], b);
  }
  uint4 o;
  o.x = __builtin_bit_cast(uint32_t, __floats2half2_rn(x[0], x[1]));
  o.y = __builtin_bit_cast(uint32_t, __floats2half2_rn(x[2], x[3]));
  o.z = __builtin_bit_cast(uint32_t, __floats2half2_rn(x[4], x[5]));
  o.w = __builtin_bit_cast(uint32_t, __floats2half2_rn(x[6], x[7]));
  return o;
}

// K: lane (position, word w) handles elements 8 w .. 8 w + 7 of one
// position.  V (codes stored in position pairs: 32-bit word u of a pair
// holds dims 4u .. 4u + 3 of the even slot in its low half and of the odd
// slot in its high half): lane (pair, v) reads words 2v, 2v + 1 of a pair (8
// bytes) and handles elements 8 v .. 8 v + 7 of both positions.
template <int D, int G, bool V>
__global__ __launch_bounds__(64 * kWaves) void reconstruct_kernel(
    const uint32_t* __restrict__ codes, const uint32_t* __restrict__ meta,
    const int32_t* __restrict__ table, int n, int kv0, int Hkv, int P, int NP,
    uint4* __restrict__ out) {
  constexpr int WPP = D / 8;         // 16-byte output chunks per position
  constexpr int LPU = 64 / WPP;      // units (positions or pairs) per wave and load
  constexpr int NG = D / G;          // groups per position
  constexpr int PER = V ? 2 : 1;     // positions per unit
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int j = blockIdx.y;          // head within the group
  const int kv = kv0 + j;
  const int w = lane % WPP;
  const int g = (8 * w) / G;
  const int u0 = (blockIdx.x * kWaves + wave) * kIters * LPU + lane / WPP;

  uint32_t cw[kIters][PER], mw[kIters][PER];
#pragma unroll
  for (int i = 0; i < kIters; ++i) {
    const int t = PER * (u0 + i * LPU);  // first position of the unit
#pragma unroll
    for (int e = 0; e < PER; ++e) cw[i][e] = mw[i][e] = 0u;  // outside the pool: zeros
    const int page = t < n ? table[t / P] : -1;
    if ((unsigned)page < (unsigned)NP) {
      const size_t vec = ((size_t)page * Hkv + kv) * P + (t % P);
      if constexpr (V) {
        const uint2 c2 = *reinterpret_cast<const uint2*>(codes + vec * (D / 8) + 2 * w);
        cw[i][0] = (c2.x & 0xFFFFu) | (c2.y << 16);
        cw[i][1] = (c2.x >> 16) | (c2.y & 0xFFFF0000u);
        mw[i][0] = meta[vec * NG + g];
        mw[i][1] = meta[(vec + 1) * NG + g];
      } else {
        cw[i][0] = codes[vec * WPP + w];
        mw[i][0] = meta[vec * NG + g];
      }
    }
  }
#pragma unroll
  for (int i = 0; i < kIters; ++i) {
    const int t = PER * (u0 + i * LPU);
#pragma unroll
    for (int e = 0; e < PER; ++e) {
      const uint4 o = emit8(cw[i][e], mw[i][e]);
      if (t + e < n) out[((size_t)j * n + t + e) * WPP + w] = o;
    }
  }
}

template <int D, int G>
hipError_t launch_t(const jf_kv_layout& L, const jf_kv_pool_ptrs& pool, const int32_t* table,
                    int32_t n, int32_t kv0, int32_t g, void* k_out, void* v_out,
                    hipStream_t stream) {
  constexpr int LPU = 64 / (D / 8);
  constexpr int kUnits = kWaves * kIters * LPU;  // units per block
  const unsigned kb = (unsigned)((n + kUnits - 1) / kUnits);
  const unsigned vb = (unsigned)((n + 2 * kUnits - 1) / (2 * kUnits));
  hipLaunchKernelGGL((reconstruct_kernel<D, G, false>), dim3(kb, (unsigned)g), dim3(64 * kWaves),
                     0, stream, static_cast<const uint32_t*>(pool.k_codes),
                     static_cast<const uint32_t*>(pool.k_meta), table, n, kv0, L.num_kv_heads,
                     L.page_size, L.num_pages, static_cast<uint4*>(k_out));
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((reconstruct_kernel<D, G, true>), dim3(vb, (unsigned)g), dim3(64 * kWaves),
                     0, stream, static_cast<const uint32_t*>(pool.v_codes),
                     static_cast<const uint32_t*>(pool.v_meta), table, n, kv0, L.num_kv_heads,
                     L.page_size, L.num_pages, static_cast<uint4*>(v_out));
  return hipGetLastError();
}

}  // namespace

namespace jfkv {

hipError_t launch_reconstruct(const jf_kv_layout& L, const jf_kv_pool_ptrs& pool,
                              const int32_t* block_table, int32_t max_pages, int32_t n_pos,
                              int32_t kv0, int32_t num_heads, void* k_out, void* v_out,
                              hipStream_t stream) {
  if (n_pos == 0) return hipSuccess;
#define JF_CASE(D_, G_)                                                                     \
  if (L.head_dim == D_ && L.group_size == G_)                                               \
    return launch_t<D_, G_>(L, pool, block_table, n_pos, kv0, num_heads, k_out, v_out, stream);
  JF_CASE(64, 32)
  JF_CASE(64, 64)
  JF_CASE(128, 32)
  JF_CASE(128, 64)
  JF_CASE(128, 128)
  JF_CASE(256, 32)
  JF_CASE(256, 64)
  JF_CASE(256, 128)
#undef JF_CASE
  return hipErrorInvalidValue;
}

}  // namespace jfkv
