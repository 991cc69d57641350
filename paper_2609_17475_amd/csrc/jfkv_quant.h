// Device-side quantizer of one group (the contract in include/jfkv.h),
// shared by the append kernels and the fused decode step.  Every binary32
// step is a separately rounded IEEE operation (explicit _rn intrinsics; no
// contraction applies).
#pragma once

#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>

#include <cstdint>

namespace jfkv {

// Monotone unsigned key of an fp16 bit pattern (-0 below +0; finite values).
__device__ __forceinline__ uint32_t q_order_key(uint32_t h) {
  return (h & 0x8000u) ? (~h & 0xffffu) : (h | 0x8000u);
}
__device__ __forceinline__ uint32_t q_from_key(uint32_t k) {
  return (k & 0x8000u) ? (k & 0x7fffu) : (~k & 0xffffu);
}

__device__ __forceinline__ float q_h2f(uint32_t bits) {
  return __half2float(__ushort_as_half((unsigned short)bits));
}

// fp16 of a positive binary32 value, rounded toward +inf: round to nearest
// even, then step up one ulp if that fell below.
__device__ __forceinline__ uint32_t q_f2h_up_pos(float x) {
  uint32_t h = __half_as_ushort(__float2half_rn(x));
  if (q_h2f(h) < x) h += 1;  // positive patterns are ordered like their values
  return h;
}

// One lane's share of quantizing a group: the lane holds 8 consecutive fp16
// values (element i in half i % 2 of word i / 2) of a group spread over
// `lpg` consecutive lanes, lpg-aligned.  Every lane of the wave must call
// this (the group's minimum and maximum are exchanged by lane swaps).
// Returns the 8 codes packed as nibbles (element i at bits 4i..4i+3) and the
// group's (scale | bias << 16) fp16 word.
__device__ __forceinline__ uint32_t quantize8(uint4 x, int lpg, uint32_t& meta_word) {
  const uint32_t w[4] = {x.x, x.y, x.z, x.w};
  uint32_t kmin = 0xffffu, kmax = 0u;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const uint32_t k0 = q_order_key(w[i] & 0xffffu), k1 = q_order_key(w[i] >> 16);
    kmin = min(kmin, min(k0, k1));
    kmax = max(kmax, max(k0, k1));
  }
  for (int off = 1; off < lpg; off <<= 1) {
    kmin = min(kmin, (uint32_t)__shfl_xor((int)kmin, off));
    kmax = max(kmax, (uint32_t)__shfl_xor((int)kmax, off));
  }
  const uint32_t mn_bits = q_from_key(kmin), mx_bits = q_from_key(kmax);
  const float mn = q_h2f(mn_bits), mx = q_h2f(mx_bits);
  // bias: fp16 of mn rounded toward -inf; mn is an fp16 value, so exact
  const uint32_t bias_bits = mn_bits;
  const float range = __fsub_rn(mx, mn);
  const float step = __fdiv_rn(range, 15.0f);
  const uint32_t scale_bits = (range == 0.0f) ? 0u : q_f2h_up_pos(step);
  const float sf = q_h2f(scale_bits), bf = q_h2f(bias_bits);
  uint32_t packed = 0;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    uint32_t code = 0;
    if (scale_bits != 0) {
      const float xi = q_h2f((w[i >> 1] >> ((i & 1) * 16)) & 0xffffu);
      const float r = __fdiv_rn(__fsub_rn(xi, bf), sf);
      float qf = __builtin_rintf(r);
      qf = fminf(fmaxf(qf, 0.0f), 15.0f);
      code = (uint32_t)qf;
    }
    packed |= code << (4 * i);
  }
  meta_word = scale_bits | (bias_bits << 16);
  return packed;
}

// Store one lane's 8 codes (dims 8 c8 .. 8 c8 + 7 of a vector) at position
// `slot` of the (page, KV head) run `ph` = page * Hkv + kv, and its group's
// (scale, bias) word from the group's first lane (c8 % lpg == 0).  K rows:
// one 32-bit word; V (position-paired layout): the slot's 16-bit halves of
// the pair words of 4-dim chunks 2 c8 and 2 c8 + 1, leaving the other
// position's halves as they are.
__device__ __forceinline__ void store_codes8(uint8_t* codes, uint32_t* meta, bool is_v,
                                             int64_t ph, int P, int D, int G, int slot, int c8,
                                             int lpg, uint32_t packed, uint32_t meta_word) {
  if (!is_v) {
    uint32_t* dst = reinterpret_cast<uint32_t*>(codes + (ph * P + slot) * (D / 2)) + c8;
    *dst = packed;
  } else {
    uint16_t* base = reinterpret_cast<uint16_t*>(codes + ph * P * (D / 2) +
                                                 ((int64_t)(slot >> 1) * (D / 4) + 2 * c8) * 4 +
                                                 (slot & 1) * 2);
    base[0] = (uint16_t)(packed & 0xffffu);
    base[2] = (uint16_t)(packed >> 16);
  }
  if ((c8 % lpg) == 0) meta[(ph * P + slot) * (D / G) + (c8 * 8) / G] = meta_word;
}

}  // namespace jfkv
