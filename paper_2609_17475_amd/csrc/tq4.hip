// TQ4 encode-and-append: each 256-element K or V vector is divided by its
// norm, rotated by H_256 S / 16 (unnormalised Hadamard matrix H_256, random
// signs S) and every rotated coordinate replaced by the index of one of 16
// shared centroids (Sec. 3.1, eq. codec).  The indices are packed eight per
// u32 word and stored with the fp16 norm at the vector's page slot
// (Appendix A, Table codec; Background, page table).
//
// One wave per vector at a time, eight vectors per wave (their loads issued
// together).  Lane l holds elements 4l .. 4l + 3 (one 8-byte load: the 64
// lanes read the vector's 512 bytes in one coalesced access).  The
// Walsh-Hadamard transform takes the first two of its eight butterfly stages
// inside each lane (element index bits 0 and 1) and the other six across
// lanes (index bits 2..7 are lane bits 0..5), with one exchange per stage and
// value (DPP, swizzle or lane permute: no LDS addresses).  The norm is a wave-wide sum of squares: IEEE addition commutes, so
// every lane of the butterfly reduction ends with the same sum.
//
// Index of a coordinate: the number of midpoint thresholds between adjacent
// centroids that it strictly exceeds (a coordinate on a threshold keeps the
// lower index), over the float32 midpoints (c_j + c_{j+1}) / 2.  It is read
// from a table of 64 buckets of the coordinate range: the bucket map
// floor(y / w + o), clamped, is monotone, so every threshold whose own
// bucket is lower lies below y and every one in a higher bucket above it;
// an entry holds the count of thresholds in lower buckets and the one
// threshold of its bucket (+inf if none), and the index is that count plus
// one comparison.  If a codebook puts two thresholds in one bucket, the block
// uses a 4-step binary search over the midpoints instead.  Both give the
// same index for every y.  y is the transformed vector times one correctly
// rounded reciprocal of 16 rho.
//
// The destination of a row (request, logical position, page) is looked up
// once per row: a wave's vectors are consecutive, Hkv of them per row.
// A vector of norm 0 has every coordinate 0.
#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "jfkv.h"
#include "jfkv_internal.h"

namespace {

constexpr int kD = 256;          // head dimension of the format
constexpr int kWavesPerBlock = 4;
constexpr int kVecPerWave = 8;   // vectors per wave, their loads issued together
constexpr int kLevels = 16;
constexpr int kBuckets = 64;     // index buckets (at most one threshold each)

__device__ __forceinline__ float2 h2_to_f2(uint32_t u) {
  return __half22float2(__builtin_bit_cast(__half2, u));
}

// The value of lane ^ M (M = 1 .. 32) of the same wave: a DPP quad
// permutation for M = 1, 2 (a VALU move), a bit-mask swizzle within each
// 32-lane half for M = 4, 8, 16, a lane permute for M = 32.
template <int M>
__device__ __forceinline__ float xor_lane(float v) {
  const int i = __builtin_bit_cast(int, v);
  if constexpr (M == 1)
    return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(i, 0xB1, 0xF, 0xF, true));
  else if constexpr (M == 2)
    return __builtin_bit_cast(float, __builtin_amdgcn_mov_dpp(i, 0x4E, 0xF, 0xF, true));
  else if constexpr (M < 32)
    return __builtin_bit_cast(float, __builtin_amdgcn_ds_swizzle(i, (M << 10) | 0x1F));
  else
    return __shfl_xor(v, M, 64);
}

// One cross-lane butterfly stage on lane bit log2(M): the lane with the bit
// set takes partner - own, the other own + partner (an fma by +-1 is exact).
template <int M>
__device__ __forceinline__ void stage(float& e0, float& e1, float& e2, float& e3, int lane) {
  const float sg = (lane & M) ? -1.0f : 1.0f;
  const float p0 = xor_lane<M>(e0), p1 = xor_lane<M>(e1);
  const float p2 = xor_lane<M>(e2), p3 = xor_lane<M>(e3);
  e0 = fmaf(sg, e0, p0);
  e1 = fmaf(sg, e1, p1);
  e2 = fmaf(sg, e2, p2);
  e3 = fmaf(sg, e3, p3);
}

__global__ __launch_bounds__(64 * kWavesPerBlock) void tq4_encode_kernel(
    uint32_t* __restrict__ words, __half* __restrict__ norms, const uint2* __restrict__ x,
    const float* __restrict__ signs, const float* __restrict__ centroids,
    const int32_t* __restrict__ cu_tok, const int32_t* __restrict__ start_pos,
    const int32_t* __restrict__ block_tables, int B, int max_pages, int Hkv, int P, int NP,
    int n_vec) {
  // thresholds for a 4-step binary search: entry 15 is +inf (never passed)
  __shared__ float thr[kLevels];
  // bucket table: y falls in bucket b = clamp(floor(fma(y, bk_inv, bk_off)),
  // 0, kBuckets - 1), a monotone map, so every threshold in a lower bucket is
  // below y and every one in a higher bucket above it; entry b holds their
  // count (below) and the bucket's own threshold (+inf if none)
  __shared__ float2 bucket[kBuckets];
  __shared__ int s_multi;  // a bucket holds two thresholds: binary search instead
  if (threadIdx.x < kLevels)
    thr[threadIdx.x] = threadIdx.x < kLevels - 1
                           ? (centroids[threadIdx.x] + centroids[threadIdx.x + 1]) * 0.5f
                           : INFINITY;
  if (threadIdx.x == 0) s_multi = 0;
  __syncthreads();
  // buckets of width (t_14 - t_0) / (kBuckets - 2) from one width below t_0
  const float t_first = thr[0], t_last = thr[kLevels - 2];
  const float bk_inv = (float)(kBuckets - 2) / (t_last - t_first);
  const float bk_off = 1.0f - t_first * bk_inv;
  auto bucket_of = [&](float y) {  // (clamped before the conversion: no overflow)
    return (int)__builtin_amdgcn_fmed3f(fmaf(y, bk_inv, bk_off), 0.0f, (float)(kBuckets - 1));
  };
  if (threadIdx.x < kBuckets) {
    int below = 0, inside = 0;
    float t_in = INFINITY;
    for (int k = 0; k < kLevels - 1; ++k) {
      const int bt = bucket_of(thr[k]);
      below += bt < (int)threadIdx.x;
      if (bt == (int)threadIdx.x) {
        ++inside;
        t_in = thr[k];
      }
    }
    bucket[threadIdx.x] = make_float2(__builtin_bit_cast(float, below), t_in);
    if (inside > 1 || !(bk_inv > 0.0f) || !isfinite(bk_inv)) s_multi = 1;  // benign race: all write 1
  }
  __syncthreads();
  const bool use_buckets = s_multi == 0;  // block-uniform

  const int lane = threadIdx.x & 63;
  // wave-uniform from here to the stores: the vector, its request, page and
  // slot are scalar values (the host bounds n_vec by INT32_MAX)
  const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
  const int vec0 = ((int)blockIdx.x * kWavesPerBlock + wave) * kVecPerWave;
  if (vec0 >= n_vec) return;  // the whole wave
  const int nv = min(kVecPerWave, n_vec - vec0);

  const uint64_t* xw = reinterpret_cast<const uint64_t*>(x);
  uint64_t raw[kVecPerWave];
#pragma unroll
  for (int v = 0; v < kVecPerWave; ++v)
    if (v < nv) raw[v] = __builtin_nontemporal_load(&xw[(int64_t)(vec0 + v) * (kD / 4) + lane]);
  const float4 s = reinterpret_cast<const float4*>(signs)[lane];
  int row_cur = vec0 / Hkv, kv_cur = vec0 - row_cur * Hkv;  // of the next vector
  int row_done = -1, page_row = -1, slot_in_page = 0;       // the looked-up row

#pragma unroll
  for (int v = 0; v < kVecPerWave; ++v) {
    if (v >= nv) break;
    const float2 f01 = h2_to_f2((uint32_t)raw[v]), f23 = h2_to_f2((uint32_t)(raw[v] >> 32));

    // norm: squares of fp16 values are exact in float32
    float ss = f01.x * f01.x + f01.y * f01.y + f23.x * f23.x + f23.y * f23.y;
    ss += xor_lane<32>(ss);
    ss += xor_lane<16>(ss);
    ss += xor_lane<8>(ss);
    ss += xor_lane<4>(ss);
    ss += xor_lane<2>(ss);
    ss += xor_lane<1>(ss);
    const float rho = sqrtf(ss);

    // H_256 S x: two stages in the lane, six across lanes
    float e0 = s.x * f01.x, e1 = s.y * f01.y, e2 = s.z * f23.x, e3 = s.w * f23.y;
    {
      const float a0 = e0 + e1, a1 = e0 - e1, a2 = e2 + e3, a3 = e2 - e3;
      e0 = a0 + a2; e1 = a1 + a3; e2 = a0 - a2; e3 = a1 - a3;
    }
    stage<1>(e0, e1, e2, e3, lane);
    stage<2>(e0, e1, e2, e3, lane);
    stage<4>(e0, e1, e2, e3, lane);
    stage<8>(e0, e1, e2, e3, lane);
    stage<16>(e0, e1, e2, e3, lane);
    stage<32>(e0, e1, e2, e3, lane);
    // rotated unit vector y = H S x / (16 rho), by one rounded reciprocal
    const float inv = rho > 0.0f ? __fdiv_rn(1.0f, rho * 16.0f) : 0.0f;
    const float y[4] = {e0 * inv, e1 * inv, e2 * inv, e3 * inv};

    uint32_t q = 0;  // four 4-bit indices: element 4 lane + j at bits 4j
    if (use_buckets) {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const float2 e = bucket[bucket_of(y[j])];
        const int idx = __builtin_bit_cast(int, e.x) + (y[j] > e.y ? 1 : 0);
        q |= (uint32_t)idx << (4 * j);
      }
    } else {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      // off = 4 x the number of thresholds strictly below y[j] found so far
      // (a byte offset, so each level's read takes its constant part as the
      // instruction's offset)
      int off = 0;
#pragma unroll
      for (int step = 8; step >= 1; step >>= 1) {
        const float t = *reinterpret_cast<const float*>(reinterpret_cast<const char*>(thr) + off +
                                                        4 * (step - 1));
        off += y[j] > t ? 4 * step : 0;
      }
      q |= (uint32_t)(off >> 2) << (4 * j);
    }
    }
    // word w = elements 8w .. 8w + 7: lanes 2w (low half) and 2w + 1
    const uint32_t partner = __builtin_bit_cast(uint32_t, xor_lane<1>(__builtin_bit_cast(float, q)));
    const uint32_t word = q | (partner << 16);

    // (row, kv) of this vector; the row's destination is looked up once per
    // row (the vectors of a wave are consecutive: Hkv of them per row)
    const int kv = kv_cur;
    if (++kv_cur == Hkv) kv_cur = 0;
    if (row_cur != row_done) {
      row_done = row_cur;
      int32_t lo = 0, hi = B;  // request: largest b with cu_tok[b] <= row
      while (hi - lo > 1) {
        const int32_t mid = (lo + hi) >> 1;
        if (cu_tok[mid] <= row_cur) lo = mid; else hi = mid;
      }
      const int64_t pos = (int64_t)start_pos[lo] + (row_cur - cu_tok[lo]);
      page_row = -1;
      if (pos >= 0 && pos < (int64_t)max_pages * P) {
        const int lp = (int)pos / P;
        page_row = block_tables[(int64_t)lo * max_pages + lp];
        slot_in_page = (int)pos - lp * P;
      }
    }
    if (kv_cur == 0) ++row_cur;
    if (page_row < 0 || page_row >= NP) continue;
    const int64_t slot = ((int64_t)page_row * Hkv + kv) * P + slot_in_page;
    if ((lane & 1) == 0) words[slot * (kD / 8) + (lane >> 1)] = word;
    if (lane == 0) norms[slot] = __float2half_rn(rho);
  }
}

// Page -> operand reconstruction of TQ4 vectors (Appendix A, Table codec:
// page lookup, index unpacking, centroid lookup, inverse rotation, norm
// restoration in one kernel): x_hat = rho_hat S H_256 c[z] / 16 for KV heads
// kv0 .. kv0 + g - 1 at logical positions 0 .. n - 1 of one request, written
// as contiguous fp16 [g][n][256] K (blockIdx.z = 0) or V operands.  One wave
// per vector, kVecPerWave vectors per wave with their loads issued together;
// lane l holds elements 4l .. 4l + 3 (its half of index word l / 2), looks
// their centroids up in LDS and runs the same eight butterfly stages as the
// encoder (H_256 is symmetric), then multiplies by its signs and rho_hat / 16
// (fp32) and writes 8 bytes, so a vector's 512 bytes leave in one coalesced
// store.  A page ID outside the pool gives zeros.
__global__ __launch_bounds__(64 * kWavesPerBlock) void tq4_reconstruct_kernel(
    const uint32_t* __restrict__ k_words, const __half* __restrict__ k_norms,
    const uint32_t* __restrict__ v_words, const __half* __restrict__ v_norms,
    const float* __restrict__ k_signs, const float* __restrict__ v_signs,
    const float* __restrict__ centroids, const int32_t* __restrict__ table, int n, int kv0,
    int Hkv, int P, int NP, uint2* __restrict__ k_out, uint2* __restrict__ v_out) {
  __shared__ float cent[kLevels];
  if (threadIdx.x < kLevels) cent[threadIdx.x] = centroids[threadIdx.x];
  __syncthreads();
  const bool is_v = blockIdx.z != 0;
  const uint32_t* words = is_v ? v_words : k_words;
  const __half* norms = is_v ? v_norms : k_norms;
  uint2* out = is_v ? v_out : k_out;
  const int j = blockIdx.y;
  const int kv = kv0 + j;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
  const int t0 = ((int)blockIdx.x * kWavesPerBlock + wave) * kVecPerWave;
  if (t0 >= n) return;  // the whole wave
  const int nv = min(kVecPerWave, n - t0);
  const float4 sg = reinterpret_cast<const float4*>(is_v ? v_signs : k_signs)[lane];

  uint32_t wd[kVecPerWave];
  float rho[kVecPerWave];
  bool ok[kVecPerWave];
#pragma unroll
  for (int v = 0; v < kVecPerWave; ++v) {
    wd[v] = 0u;
    rho[v] = 0.0f;
    ok[v] = false;  // outside the pool: zeros
    if (v < nv) {
      const int t = t0 + v;
      const int page = table[t / P];  // wave-uniform
      ok[v] = (unsigned)page < (unsigned)NP;
      if (ok[v]) {
        const int64_t vec = ((int64_t)page * Hkv + kv) * P + (t % P);
        wd[v] = words[vec * (kD / 8) + (lane >> 1)];
        rho[v] = __half2float(norms[vec]);
      }
    }
  }
#pragma unroll
  for (int v = 0; v < kVecPerWave; ++v) {
    if (v >= nv) break;
    const uint32_t q = wd[v] >> (16 * (lane & 1));  // element 4 lane + i at bits 4 i
    float e0 = cent[q & 15u], e1 = cent[(q >> 4) & 15u];
    float e2 = cent[(q >> 8) & 15u], e3 = cent[(q >> 12) & 15u];
    {
      const float a0 = e0 + e1, a1 = e0 - e1, a2 = e2 + e3, a3 = e2 - e3;
      e0 = a0 + a2; e1 = a1 + a3; e2 = a0 - a2; e3 = a1 - a3;
    }
    stage<1>(e0, e1, e2, e3, lane);
    stage<2>(e0, e1, e2, e3, lane);
    stage<4>(e0, e1, e2, e3, lane);
    stage<8>(e0, e1, e2, e3, lane);
    stage<16>(e0, e1, e2, e3, lane);
    stage<32>(e0, e1, e2, e3, lane);
    const float f = rho[v] * 0.0625f;
    uint2 o = make_uint2(0u, 0u);
    if (ok[v]) {
      o.x = __builtin_bit_cast(uint32_t, __floats2half2_rn(sg.x * e0 * f, sg.y * e1 * f));
      o.y = __builtin_bit_cast(uint32_t, __floats2half2_rn(sg.z * e2 * f, sg.w * e3 * f));
    }
    out[((int64_t)j * n + t0 + v) * (kD / 4) + lane] = o;
  }
}

}  // namespace

namespace jfkv {

hipError_t launch_tq4_reconstruct(const jf_kv_layout& L, const void* k_words, const void* k_norms,
                                  const void* v_words, const void* v_norms, const float* k_signs,
                                  const float* v_signs, const float* centroids,
                                  const int32_t* block_table, int32_t n_pos, int32_t kv0,
                                  int32_t num_heads, void* k_out, void* v_out,
                                  hipStream_t stream) {
  if (n_pos == 0) return hipSuccess;
  constexpr int kPerBlock = kWavesPerBlock * kVecPerWave;
  dim3 grid((unsigned)((n_pos + kPerBlock - 1) / kPerBlock), (unsigned)num_heads, 2);
  hipLaunchKernelGGL(tq4_reconstruct_kernel, grid, dim3(64 * kWavesPerBlock), 0, stream,
                     static_cast<const uint32_t*>(k_words), static_cast<const __half*>(k_norms),
                     static_cast<const uint32_t*>(v_words), static_cast<const __half*>(v_norms),
                     k_signs, v_signs, centroids, block_table, n_pos, kv0, L.num_kv_heads,
                     L.page_size, L.num_pages, static_cast<uint2*>(k_out),
                     static_cast<uint2*>(v_out));
  return hipGetLastError();
}

hipError_t launch_tq4_encode(const jf_kv_layout& L, void* words, void* norms, const void* x,
                             const float* signs, const float* centroids, const int32_t* cu_tok,
                             const int32_t* start_pos, const int32_t* block_tables, int32_t B,
                             int32_t max_pages, int32_t total_tok, hipStream_t stream) {
  const int64_t n_vec = (int64_t)total_tok * L.num_kv_heads;
  constexpr int kPerBlock = kWavesPerBlock * kVecPerWave;
  const int64_t blocks = (n_vec + kPerBlock - 1) / kPerBlock;
  if (n_vec > 0x7fffffffLL) return hipErrorInvalidValue;
  hipLaunchKernelGGL(tq4_encode_kernel, dim3((unsigned)blocks), dim3(64 * kWavesPerBlock), 0,
                     stream, static_cast<uint32_t*>(words), static_cast<__half*>(norms),
                     static_cast<const uint2*>(x), signs, centroids, cu_tok, start_pos,
                     block_tables, B, max_pages, L.num_kv_heads, L.page_size, L.num_pages,
                     (int)n_vec);
  return hipGetLastError();
}

}  // namespace jfkv
