// TQ4 encode-and-append: each 256-element K or V vector is divided by its
// norm, rotated by H_256 S / 16 (unnormalised Hadamard matrix H_256, random
// signs S) and every rotated coordinate replaced by the index of one of 16
// shared centroids (Sec. 3.1, eq. codec).  The indices are packed eight per
// u32 word and stored with the fp16 norm at the vector's page slot
// (Appendix A, Table codec; Background, page table).
//
// One wave per vector.  Lane l holds elements 4l .. 4l + 3 (one 8-byte load:
// the 64 lanes read the vector's 512 bytes in one coalesced access).  The
// Walsh-Hadamard transform takes the first two of its eight butterfly stages
// inside each lane (element index bits 0 and 1) and the other six across
// lanes (index bits 2..7 are lane bits 0..5), with one exchange per stage and
// value.  The norm is a wave-wide sum of squares: IEEE addition commutes, so
// every lane of the butterfly reduction ends with the same sum.
//
// Index of a coordinate: the number of midpoint thresholds between adjacent
// centroids that it strictly exceeds (a coordinate on a threshold keeps the
// lower index).  The thresholds are the float32 midpoints (c_j + c_{j+1}) / 2.
// A vector of norm 0 has every coordinate 0.
#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "jfkv.h"
#include "jfkv_internal.h"

namespace {

constexpr int kD = 256;          // head dimension of the format
constexpr int kWavesPerBlock = 4;
constexpr int kLevels = 16;

__device__ __forceinline__ float2 h2_to_f2(uint32_t u) {
  return __half22float2(__builtin_bit_cast(__half2, u));
}

__global__ __launch_bounds__(64 * kWavesPerBlock) void tq4_encode_kernel(
    uint32_t* __restrict__ words, __half* __restrict__ norms, const uint2* __restrict__ x,
    const float* __restrict__ signs, const float* __restrict__ centroids,
    const int32_t* __restrict__ cu_tok, const int32_t* __restrict__ start_pos,
    const int32_t* __restrict__ block_tables, int B, int max_pages, int Hkv, int P, int NP,
    int64_t n_vec) {
  const int lane = threadIdx.x & 63;
  const int64_t vec = (int64_t)blockIdx.x * kWavesPerBlock + (threadIdx.x >> 6);
  if (vec >= n_vec) return;  // the whole wave: one vector per wave
  const int64_t row = vec / Hkv;
  const int kv = (int)(vec - row * Hkv);

  const uint2 raw = x[vec * (kD / 4) + lane];
  const float4 s = reinterpret_cast<const float4*>(signs)[lane];
  const float2 f01 = h2_to_f2(raw.x), f23 = h2_to_f2(raw.y);

  // norm: squares of fp16 values are exact in float32
  float ss = f01.x * f01.x + f01.y * f01.y + f23.x * f23.x + f23.y * f23.y;
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) ss += __shfl_xor(ss, m, 64);
  const float rho = sqrtf(ss);

  // H_256 S x: two stages in the lane, six across lanes
  float v0 = s.x * f01.x, v1 = s.y * f01.y, v2 = s.z * f23.x, v3 = s.w * f23.y;
  {
    const float a0 = v0 + v1, a1 = v0 - v1, a2 = v2 + v3, a3 = v2 - v3;
    v0 = a0 + a2; v1 = a1 + a3; v2 = a0 - a2; v3 = a1 - a3;
  }
#pragma unroll
  for (int m = 1; m < 64; m <<= 1) {
    const bool hi = (lane & m) != 0;
    const float p0 = __shfl_xor(v0, m, 64), p1 = __shfl_xor(v1, m, 64);
    const float p2 = __shfl_xor(v2, m, 64), p3 = __shfl_xor(v3, m, 64);
    v0 = hi ? p0 - v0 : v0 + p0;
    v1 = hi ? p1 - v1 : v1 + p1;
    v2 = hi ? p2 - v2 : v2 + p2;
    v3 = hi ? p3 - v3 : v3 + p3;
  }
  // rotated unit vector y = H S x / (16 rho)
  const float den = rho * 16.0f;
  float y[4] = {v0, v1, v2, v3};
#pragma unroll
  for (int j = 0; j < 4; ++j) y[j] = rho > 0.0f ? __fdiv_rn(y[j], den) : 0.0f;

  uint32_t q = 0;  // four 4-bit indices: element 4 lane + j at bits 4j
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    uint32_t idx = 0;
#pragma unroll
    for (int t = 0; t < kLevels - 1; ++t) {
      const float thr = (centroids[t] + centroids[t + 1]) * 0.5f;
      idx += y[j] > thr ? 1u : 0u;
    }
    q |= idx << (4 * j);
  }
  // word w = elements 8w .. 8w + 7: lanes 2w (low half) and 2w + 1
  const uint32_t partner = (uint32_t)__shfl_xor((int)q, 1, 64);
  const uint32_t word = q | (partner << 16);

  // request of this row and its logical position
  int32_t lo = 0, hi = B;  // largest b with cu_tok[b] <= row
  while (hi - lo > 1) {
    const int32_t mid = (lo + hi) >> 1;
    if (cu_tok[mid] <= row) lo = mid; else hi = mid;
  }
  const int64_t pos = (int64_t)start_pos[lo] + (row - cu_tok[lo]);
  if (pos < 0) return;
  const int64_t lp = pos / P;
  if (lp >= max_pages) return;
  const int32_t page = block_tables[(int64_t)lo * max_pages + lp];
  if (page < 0 || page >= NP) return;
  const int64_t slot = ((int64_t)page * Hkv + kv) * P + (pos - lp * P);
  if ((lane & 1) == 0) words[slot * (kD / 8) + (lane >> 1)] = word;
  if (lane == 0) norms[slot] = __float2half_rn(rho);
}

}  // namespace

namespace jfkv {

hipError_t launch_tq4_encode(const jf_kv_layout& L, void* words, void* norms, const void* x,
                             const float* signs, const float* centroids, const int32_t* cu_tok,
                             const int32_t* start_pos, const int32_t* block_tables, int32_t B,
                             int32_t max_pages, int32_t total_tok, hipStream_t stream) {
  const int64_t n_vec = (int64_t)total_tok * L.num_kv_heads;
  const int64_t blocks = (n_vec + kWavesPerBlock - 1) / kWavesPerBlock;
  if (blocks > 0x7fffffffLL) return hipErrorInvalidValue;
  hipLaunchKernelGGL(tq4_encode_kernel, dim3((unsigned)blocks), dim3(64 * kWavesPerBlock), 0,
                     stream, static_cast<uint32_t*>(words), static_cast<__half*>(norms),
                     static_cast<const uint2*>(x), signs, centroids, cu_tok, start_pos,
                     block_tables, B, max_pages, L.num_kv_heads, L.page_size, L.num_pages, n_vec);
  return hipGetLastError();
}

}  // namespace jfkv
