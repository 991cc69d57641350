// Quantize-and-append of new K/V rows into 4-bit pages (gfx950).
//
// Encoding: group-wise affine 4-bit codes with an fp16 scale and bias per
// group of head_dim elements (the affine 4-bit format the paper's
// Introduction describes for weights), written into 256-token pages
// through the request's page table (Background, "Compact histories need
// reusable storage").  The contract is bit-exact; every binary32 step is a
// separately rounded IEEE operation in the order given in include/jfkv.h.
//
// Mapping: one group of G elements is handled by G/8 consecutive lanes, each
// holding 8 fp16 values (one 16-byte load), so a wave covers 8 groups (G=64)
// and a wave's loads of a K or V row segment are contiguous.  Min and max
// reduce over the group's lanes with cross-lane swaps on integer total-order
// keys of the fp16 bit patterns (exact and independent of order).  Each lane
// packs its 8 codes into one 32-bit word: one store for the row-major K
// layout, two 16-bit stores for the position-paired V layout.
#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>

#include "jfkv_internal.h"

#pragma clang fp contract(off)

namespace {

// Monotone unsigned key of an fp16 bit pattern (-0 below +0; finite values).
__device__ __forceinline__ uint32_t order_key(uint32_t h) {
  return (h & 0x8000u) ? (~h & 0xffffu) : (h | 0x8000u);
}
__device__ __forceinline__ uint32_t from_key(uint32_t k) {
  return (k & 0x8000u) ? (k & 0x7fffu) : (~k & 0xffffu);
}

__device__ __forceinline__ float h2f(uint32_t bits) {
  return __half2float(__ushort_as_half((unsigned short)bits));
}

// fp16 of a positive binary32 value, rounded toward +inf: round to nearest
// even, then step up one ulp if that fell below.
__device__ __forceinline__ uint32_t f2h_up_pos(float x) {
  uint32_t h = __half_as_ushort(__float2half_rn(x));
  if (h2f(h) < x) h += 1;  // positive patterns are ordered like their values
  return h;
}

__global__ __launch_bounds__(256) void quantize_append_kernel(
    uint8_t* __restrict__ k_codes, uint32_t* __restrict__ k_meta,
    uint8_t* __restrict__ v_codes, uint32_t* __restrict__ v_meta,
    const uint4* __restrict__ k_new, const uint4* __restrict__ v_new,
    const int32_t* __restrict__ cu_tok, const int32_t* __restrict__ start_pos,
    const int32_t* __restrict__ block_tables, int32_t B, int32_t max_pages, int32_t total_tok,
    int32_t P, int32_t Hkv, int32_t D, int32_t G, int32_t NP) {
  // work layout: [row][K|V][kv][D/8 lanes]; a lane owns dims 8c..8c+7
  const int32_t lanes_per_row_kind = Hkv * (D / 8);
  const int64_t gid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t total = (int64_t)total_tok * 2 * lanes_per_row_kind;
  const bool active = gid < total;
  int32_t row = 0, kind = 0, rem = 0;
  if (active) {
    row = (int32_t)(gid / (2 * lanes_per_row_kind));
    int32_t r2 = (int32_t)(gid % (2 * lanes_per_row_kind));
    kind = r2 / lanes_per_row_kind;
    rem = r2 % lanes_per_row_kind;
  }
  const int32_t kv = rem / (D / 8);
  const int32_t c8 = rem % (D / 8);  // 8-dim chunk within the head
  const int32_t lpg = G / 8;         // lanes per group (4, 8 or 16)

  uint4 x = make_uint4(0, 0, 0, 0);
  if (active) x = (kind ? v_new : k_new)[(int64_t)row * (Hkv * D / 8) + kv * (D / 8) + c8];
  const uint32_t w[4] = {x.x, x.y, x.z, x.w};

  uint32_t kmin = 0xffffu, kmax = 0u;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    uint32_t k0 = order_key(w[i] & 0xffffu), k1 = order_key(w[i] >> 16);
    kmin = min(kmin, min(k0, k1));
    kmax = max(kmax, max(k0, k1));
  }
  // reduce over the lpg lanes of the group (aligned runs of lpg lanes)
  for (int off = 1; off < lpg; off <<= 1) {
    kmin = min(kmin, (uint32_t)__shfl_xor((int)kmin, off));
    kmax = max(kmax, (uint32_t)__shfl_xor((int)kmax, off));
  }
  if (!active) return;

  // request of this row and its logical position
  int32_t lo = 0, hi = B;  // largest b with cu_tok[b] <= row
  while (hi - lo > 1) {
    int32_t mid = (lo + hi) >> 1;
    if (cu_tok[mid] <= row) lo = mid; else hi = mid;
  }
  const int32_t b = lo;
  const int64_t pos = (int64_t)start_pos[b] + (row - cu_tok[b]);
  if (pos < 0) return;
  const int64_t lp = pos / P;
  if (lp >= max_pages) return;
  const int32_t page = block_tables[(int64_t)b * max_pages + lp];
  if (page < 0 || page >= NP) return;
  const int32_t slot = (int32_t)(pos % P);

  const uint32_t mn_bits = from_key(kmin), mx_bits = from_key(kmax);
  const float mn = h2f(mn_bits), mx = h2f(mx_bits);
  // bias: fp16 of mn rounded toward -inf; mn is an fp16 value, so exact
  const uint32_t bias_bits = mn_bits;
  const float range = __fsub_rn(mx, mn);
  const float step = __fdiv_rn(range, 15.0f);
  const uint32_t scale_bits = (range == 0.0f) ? 0u : f2h_up_pos(step);
  const float sf = h2f(scale_bits), bf = h2f(bias_bits);

  uint32_t packed = 0;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    uint32_t code = 0;
    if (scale_bits != 0) {
      const float xi = h2f((w[i >> 1] >> ((i & 1) * 16)) & 0xffffu);
      const float r = __fdiv_rn(__fsub_rn(xi, bf), sf);
      float qf = __builtin_rintf(r);
      qf = fminf(fmaxf(qf, 0.0f), 15.0f);
      code = (uint32_t)qf;
    }
    packed |= code << (4 * i);
  }

  const int32_t g = (c8 * 8) / G;
  const int64_t ph = (int64_t)page * Hkv + kv;  // (page, kv head) block
  if (kind == 0) {
    uint32_t* dst = reinterpret_cast<uint32_t*>(k_codes + (ph * P + slot) * (D / 2)) + c8;
    *dst = packed;
  } else {
    // dims 8c..8c+3 form 4-dim chunk u = 2c, dims 8c+4..8c+7 chunk 2c+1
    uint16_t* base = reinterpret_cast<uint16_t*>(v_codes + ph * P * (D / 2) +
                                                 ((int64_t)(slot >> 1) * (D / 4) + 2 * c8) * 4 +
                                                 (slot & 1) * 2);
    base[0] = (uint16_t)(packed & 0xffffu);
    base[2] = (uint16_t)(packed >> 16);
  }
  if ((c8 % lpg) == 0) {
    uint32_t* meta = kind ? v_meta : k_meta;
    meta[(ph * P + slot) * (D / G) + g] = scale_bits | (bias_bits << 16);
  }
}

}  // namespace

namespace jfkv {

hipError_t launch_quantize_append(const jf_kv_layout& L, const jf_kv_pool_ptrs& pool,
                                  const void* k_new, const void* v_new,
                                  const int32_t* cu_tok, const int32_t* start_pos,
                                  const int32_t* block_tables, int32_t B, int32_t max_pages,
                                  int32_t total_tok, hipStream_t stream) {
  const int64_t lanes = (int64_t)total_tok * 2 * L.num_kv_heads * (L.head_dim / 8);
  const int threads = 256;
  const int64_t blocks = (lanes + threads - 1) / threads;
  if (blocks > 0x7fffffff) return hipErrorInvalidValue;
  hipLaunchKernelGGL(quantize_append_kernel, dim3((uint32_t)blocks), dim3(threads), 0, stream,
                     static_cast<uint8_t*>(pool.k_codes), static_cast<uint32_t*>(pool.k_meta),
                     static_cast<uint8_t*>(pool.v_codes), static_cast<uint32_t*>(pool.v_meta),
                     static_cast<const uint4*>(k_new), static_cast<const uint4*>(v_new), cu_tok,
                     start_pos, block_tables, B, max_pages, total_tok, L.page_size,
                     L.num_kv_heads, L.head_dim, L.group_size, L.num_pages);
  return hipGetLastError();
}

}  // namespace jfkv
