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
// a 4-bit code); converting that to fp16 rounds a second time, which differs
// from rounding the exact value only if the fp32 result was inexact.  It is
// exact whenever every sum of the group fits fp32's 24 bits: its lowest
// possible bit is that of s or of b (fp16: 10 bits below the leading one, and
// not below 2^-24; q is an integer), its highest below 2^e with 2^e above
// 15 |s| + |b|.  A group failing that test (a tiny bias under a large scale,
// or the reverse) takes the exact path: the fp32 sum's error by TwoSum
// (exact), the sum rounded to odd in fp32 (toward zero, last bit set when
// inexact), then to fp16 (rounding to odd with 13 spare bits makes the second
// rounding exact).
//
// Work: a lane reads 16 bytes of codes (32 elements) of one position (K) or
// of a pair of positions (V, stored position-paired) and their groups'
// (scale, bias) words, so a wave reads consecutive positions' codes as one
// contiguous run; each lane keeps kIters loads in flight.  The fp16 values
// of a wave's load pass (2,048 elements, 4 KiB) go through
// the wave's rows in LDS and leave as 16-byte stores of whole positions, so
// each store instruction writes 1 KiB contiguously (stored straight from the
// lanes that made them, each instruction touched a quarter of every
// position's row, and the kernel took 40 % longer).
#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "jfkv.h"
#include "jfkv_internal.h"

namespace {

constexpr int kWaves = 4;
constexpr int kIters = 2;  // 16-byte code loads in flight per lane (4: 5 % slower, 8: 10 %)

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

// Every s * q + b (q = 0 .. 15) of a group is exact in fp32 (see above).
__device__ __forceinline__ bool group_exact(float s, float b) {
  if (s == 0.0f || b == 0.0f) return true;  // one term: s * q or b, exact
  // frexp exponent e: |x| in [2^(e-1), 2^e); an fp16 value's lowest bit is
  // at 2^(e-11) or 2^-24
  const int es = __builtin_amdgcn_frexp_expf(s), eb = __builtin_amdgcn_frexp_expf(b);
  const int low = max(min(es, eb) - 11, -24);
  // one more than the bound's exponent: the rounded bound may fall below a
  // power of two the exact bound reaches
  const int high = __builtin_amdgcn_frexp_expf(fmaf(fabsf(s), 15.0f, fabsf(b))) + 1;
  return high - low <= 24;
}

// fp16 of the eight elements of one code word (element k at bits 4k) with
// the group's (scale, bias) word; the exact path for the whole wave when any
// lane's group may have inexact fp32 sums.
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
#pragma unroll
  for (int k = 0; k < 8; ++k) x[k] = fmaf(s, q[k], b);
  if (__builtin_amdgcn_ballot_w64(!group_exact(s, b)) != 0) {
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

// Lane work per load: 16 bytes of codes = 32 elements.  K: lane (position,
// c) reads code words 4c .. 4c + 3 of one position (elements 32 c .. 32 c +
// 31).  V (codes stored in position pairs: 32-bit word u of a pair holds dims
// 4u .. 4u + 3 of the even slot in its low half and of the odd slot in its
// high half): lane (pair, c) reads words 4c .. 4c + 3 of a pair, elements
// 16 c .. 16 c + 15 of both positions.  Either way the lane's elements of a
// position lie in one scale group (G >= 32) and leave as 16-byte stores.
template <int D, int G, bool V>
__device__ __forceinline__ void reconstruct_body(
    const uint4* __restrict__ codes, const uint32_t* __restrict__ meta,
    const int32_t* __restrict__ table, int n, int kv0, int Hkv, int P, int NP,
    uint4* __restrict__ out, uint4* __restrict__ xs) {
  constexpr int LPU = V ? D / 16 : D / 32;  // lanes per unit (a position, or a pair)
  constexpr int UPW = 64 / LPU;             // units per wave and load
  constexpr int PER = V ? 2 : 1;            // positions per unit
  constexpr int EPL = 32 / PER;             // elements per lane and position
  constexpr int NG = D / G;                 // groups per position
  constexpr int CPP = D / 8;                // 16-byte output chunks per position
  static_assert(G >= EPL, "a lane's elements lie in one group");
  constexpr int NPOS = UPW * PER;  // positions per load pass
  constexpr int PITCH = CPP + 1;   // 16-byte chunks per LDS row (one of padding)
  static_assert(NPOS * CPP == 256 && NPOS * PITCH == 256 + 2048 / D, "four 16-byte chunks per lane and pass");
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int j = blockIdx.y;  // head within the group
  const int kv = kv0 + j;
  const int c = lane % LPU;
  const int g = (EPL * c) / G;
  const int u0 = (blockIdx.x * kWaves + wave) * kIters * UPW + lane / LPU;

  uint4 cw[kIters];
  uint32_t mw[kIters][PER];
#pragma unroll
  for (int i = 0; i < kIters; ++i) {
    const int t = PER * (u0 + i * UPW);  // first position of the unit
    cw[i] = make_uint4(0u, 0u, 0u, 0u);
#pragma unroll
    for (int e = 0; e < PER; ++e) mw[i][e] = 0u;  // outside the pool: zeros
    const int page = t < n ? table[t / P] : -1;
    if ((unsigned)page < (unsigned)NP) {
      const size_t vec = ((size_t)page * Hkv + kv) * P + (t % P);
      // (a pair's first vector: the pair's words start at its byte offset)
      cw[i] = codes[vec * (D / 32) + c];
#pragma unroll
      for (int e = 0; e < PER; ++e) mw[i][e] = meta[(vec + e) * NG + g];
    }
  }
#pragma unroll
  for (int i = 0; i < kIters; ++i) {
    uint32_t w[PER][EPL / 8];  // K-order code words per position
    if constexpr (V) {
      const uint32_t a[4] = {cw[i].x, cw[i].y, cw[i].z, cw[i].w};
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        w[0][h] = (a[2 * h] & 0xFFFFu) | (a[2 * h + 1] << 16);
        w[1][h] = (a[2 * h] >> 16) | (a[2 * h + 1] & 0xFFFF0000u);
      }
    } else {
      w[0][0] = cw[i].x; w[0][1] = cw[i].y; w[0][2] = cw[i].z; w[0][3] = cw[i].w;
    }
    // the pass's outputs (NPOS consecutive positions) through the wave's
    // LDS rows, so that each store covers whole positions: 1 KiB contiguous
    // per store instruction
#pragma unroll
    for (int e = 0; e < PER; ++e) {
#pragma unroll
      for (int h = 0; h < EPL / 8; ++h)
        xs[(PER * (lane / LPU) + e) * PITCH + (EPL / 8) * c + h] = emit8(w[e][h], mw[i][e]);
    }
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    __builtin_amdgcn_wave_barrier();
    const int tb = PER * ((blockIdx.x * kWaves + wave) * kIters * UPW + i * UPW);
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      const int q = lane + 64 * s, pos = q / CPP, ch = q % CPP;
      const uint4 val = xs[pos * PITCH + ch];
      if (tb + pos < n) out[((size_t)j * n + tb + pos) * CPP + ch] = val;
    }
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    __builtin_amdgcn_wave_barrier();
  }
}

// K (blockIdx.z = 0) and V (1) in one launch.
template <int D, int G>
__global__ __launch_bounds__(64 * kWaves) void reconstruct_kernel(
    const uint4* __restrict__ k_codes, const uint32_t* __restrict__ k_meta,
    const uint4* __restrict__ v_codes, const uint32_t* __restrict__ v_meta,
    const int32_t* __restrict__ table, int n, int kv0, int Hkv, int P, int NP,
    uint4* __restrict__ k_out, uint4* __restrict__ v_out) {
  __shared__ uint4 xs[kWaves][256 + 2048 / D];  // 2048 / D rows of D / 8 + 1 chunks per wave
  uint4* const xw = xs[threadIdx.x >> 6];
  if (blockIdx.z == 0)
    reconstruct_body<D, G, false>(k_codes, k_meta, table, n, kv0, Hkv, P, NP, k_out, xw);
  else
    reconstruct_body<D, G, true>(v_codes, v_meta, table, n, kv0, Hkv, P, NP, v_out, xw);
}

template <int D, int G>
hipError_t launch_t(const jf_kv_layout& L, const jf_kv_pool_ptrs& pool, const int32_t* table,
                    int32_t n, int32_t kv0, int32_t g, void* k_out, void* v_out,
                    hipStream_t stream) {
  // positions per block: kWaves waves x kIters loads x (64 / lanes per
  // unit) units x positions per unit; the same for K and V
  constexpr int kPos = kWaves * kIters * 64 / (D / 32);
  const unsigned blocks = (unsigned)((n + kPos - 1) / kPos);
  hipLaunchKernelGGL((reconstruct_kernel<D, G>), dim3(blocks, (unsigned)g, 2), dim3(64 * kWaves),
                     0, stream, static_cast<const uint4*>(pool.k_codes),
                     static_cast<const uint32_t*>(pool.k_meta),
                     static_cast<const uint4*>(pool.v_codes),
                     static_cast<const uint32_t*>(pool.v_meta), table, n, kv0, L.num_kv_heads,
                     L.page_size, L.num_pages, static_cast<uint4*>(k_out),
                     static_cast<uint4*>(v_out));
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
