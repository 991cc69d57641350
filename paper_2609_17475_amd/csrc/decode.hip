// Split-K single-query decode attention over the paged 4-bit KV cache
// (gfx950; both contractions on the matrix cores).
//
// The decode kernel reads the compressed pages where they are used instead of
// expanding the cache (Sec. 3.1, "Decode and prefill need different
// kernels"); query heads share their KV head (eq. groupattention), so the
// scores of one KV head's query heads against a run of positions, and the
// value sums, are small dense products.  Work is split over page-aligned
// ranges of each request ("split-K"); each split writes an fp32 partial
// (o, m, l) and the last split of a (request, KV head) to finish merges them
// with a log-sum-exp combine, so the workspace is bounded by the split cap,
// not by the context length.
//
// Data movement: a block of waves (eight at d <= 128) owns one split; its
// waves take the split's rows (a row = 32 positions of one page) in turn and
// stream each row into a private LDS ring with global_load_lds (HBM -> LDS
// without registers), all ring stages in flight while a row is computed.
// The waves meet at a barrier once per ring cycle.
//
// Arithmetic (v_mfma_f32_16x16x32_f16, fp32 accumulation): a 4-bit code
// masked into the low bits of an fp16 half is the subnormal c * 2^-24 (a
// nibble at bits 4..7: 16 c * 2^-24), which the matrix cores take exactly,
// so one AND per pair of codes makes an operand; the scale and bias of each
// group are applied to the fp32 results:
//   scores  S^T[pos][col] = K codes [pos][dim] x Q' [dim][col]: the 16
//           columns are head slots x column slots (col = head + H * slot, H
//           head slots), column slot "slot" stands for scale group slot mod
//           (groups per 128-dim half) of its head's half, and Q' holds that
//           head's query restricted to the group's dims (zero elsewhere), so
//           every column belongs to one scale group; logit = sum over the
//           head's distinct groups of
//           (scale_g * S^T + bias_g * sum(q over g's dims)) * 2^24;
//   values  O^T[dim][col] += V codes [dim][pos] x W [pos][col] with
//           W = p * scale_g (fp16) of the group that column's slot stands
//           for, the codes again subnormal operands (16 code * 2^-24: a
//           shift and an AND per pair).
//           The value is assembled as sum W (code - 8) + sum p (bias_g +
//           8 scale_g): the centred form, because where an outlier channel
//           widens a group's range the other channels' codes sit near the
//           middle, scale * code and bias are large and of opposite sign
//           while the value is small, and the fp16 rounding of W would be
//           amplified by |scale * code| / |o| in an uncentred sum.  The
//           centring costs no operand arithmetic: sum W (code - 8) =
//           sum W code - 8 sum W with sum W taken from the same rounded W,
//           so it equals the centred sum exactly; only the fp32 accumulation
//           sees the larger uncentred partial sums (~2^-24 * 15 sum W per
//           step).  sum p * bias, and sum (p * scale - W), are accumulated
//           separately in fp32 from exact products.
// Online softmax keeps one running maximum per head; it is raised only when
// a logit exceeds it by more than 2 (log2 units), so p <= 4 and p * scale
// stays within fp16 for any scale the quantizer produces (at most 65504 * 2
// / 15), and rescaling is rare.
#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>

#include <algorithm>
#include <mutex>
#include <type_traits>

#include "jfkv_internal.h"
#include "jfkv_quant.h"

// Device scratch of the allocation-free decode step (jf_decode_step_q4_static):
// completion counters, then split records; one copy per device, held until
// the process ends.  Host code uses the address hipGetSymbolAddress returns,
// never this name.
static __device__ __align__(256) uint8_t scratch[jfkv::kStaticScratchBytes];

namespace {

typedef _Float16 h2 __attribute__((ext_vector_type(2)));
typedef _Float16 h8 __attribute__((ext_vector_type(8)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(3))) void lds_void;

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kTau = 2.0f;  // lazy-rescale margin, log2 units
// Initial running maximum: finite, so that positions masked to -inf before
// any valid one give p = 2^(-inf - kMinit) = 0, not NaN.
constexpr float kMinit = -1e30f;
constexpr int kMaxThreads = 512;    // a block: one split, one block per CU
constexpr int kRowPos = 32;         // positions per row: two 16-position MFMA tiles
constexpr int kXcds = 8;            // XCDs of the chip (block placement only)
constexpr int kRingBudget = 162816; // LDS bytes of a block's rings (a CU's LDS less 1 KiB)
// Waves per block: two per SIMD where the LDS rings fit (d <= 128), so one
// wave computes while the other waits on its page loads; the waves meet at a
// barrier once per ring cycle, which keeps the two waves of a SIMD in step
// (otherwise the older one runs ahead and the block waits for the other).
#ifndef JF_DECODE_WAVES
#define JF_DECODE_WAVES 8
#endif
#ifndef JF_DECODE_STAGES
#define JF_DECODE_STAGES 3
#endif
template <int D>
constexpr int waves_for() { return D <= 128 ? JF_DECODE_WAVES : 4; }
// Query heads per block (a head chunk): the 16 columns of the matrix-core
// products are head slots times column slots, and each column slot stands for
// one scale group of a 128-dim half, so a head needs as many columns as a
// half has groups (at least one); at most one head per wave (the combine).
template <int D, int G>
constexpr int head_slots() {
  constexpr int ngh = (D < 128 ? D : 128) / G;
  constexpr int hs = 16 / (ngh > 0 ? ngh : 1);
  return hs < waves_for<D>() ? hs : waves_for<D>();
}
constexpr int kMaxStages = JF_DECODE_STAGES;  // LDS ring depth per wave (at most)

__device__ __forceinline__ h2 as_h2(uint32_t u) { return __builtin_bit_cast(h2, u); }

// s * n + b * q + acc with s and b the low and high fp16 halves of one
// (scale, bias) word (the conversions fold into v_fma_mix).  Plain code, not
// asm: n comes straight from a matrix-core result, and only the compiler's
// hazard tracking knows how long to wait before reading it.
__device__ __forceinline__ float fold_meta(uint32_t sb, float n, float q, float acc) {
  const h2 m = as_h2(sb);
  return fmaf((float)m.x, n, fmaf((float)m.y, q, acc));
}

// v + (v of the lane N places along the same 16-lane row, cyclically).
template <int N>
__device__ __forceinline__ float row_ror_add(float v) {
  return v + __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v),
                                                                   0x120 + N, 0xF, 0xF, true));
}

// Maximum of eight finite or -inf values in four v_max3/v_max instructions
// (the compiler's IEEE maximum first quiets each operand that does not come
// from arithmetic it can see, one more instruction per value).  The inputs
// are results of ordinary vector instructions, which the hardware interlocks.
__device__ __forceinline__ float max8(float a, float b, float c, float d, float e, float f,
                                      float g, float h) {
  float x, y, z, r;
  asm("v_max3_f32 %0, %1, %2, %3" : "=v"(x) : "v"(a), "v"(b), "v"(c));
  asm("v_max3_f32 %0, %1, %2, %3" : "=v"(y) : "v"(d), "v"(e), "v"(f));
  asm("v_max3_f32 %0, %1, %2, %3" : "=v"(z) : "v"(g), "v"(h), "v"(x));
  asm("v_max_f32 %0, %1, %2" : "=v"(r) : "v"(y), "v"(z));
  return r;
}

// Lane index from a volatile instruction: code that uses it cannot be hoisted
// out of a loop, so rarely taken paths keep no lane-derived registers live.
__device__ __forceinline__ int lane_id_volatile() {
  int l;
  asm volatile("v_mbcnt_lo_u32_b32 %0, -1, 0\n\tv_mbcnt_hi_u32_b32 %0, -1, %0" : "=v"(l));
  return l;
}
__device__ __forceinline__ float shfl_xor_at(float v, int lane, int off) {
  return __builtin_bit_cast(float,
                            __builtin_amdgcn_ds_bpermute((lane ^ off) << 2, __builtin_bit_cast(int, v)));
}
// Maximum over lanes lane % from .. == const: offsets from, 2 from, ..., 32.
__device__ __forceinline__ float xor_max_from(float v, int from) {
  const int ln = lane_id_volatile();
  for (int off = from; off < 64; off <<= 1) v = fmaxf(v, shfl_xor_at(v, ln, off));
  return v;
}

// HBM -> LDS loads of the page stream: lane i's 16 (or 4) bytes at
// sbase + voff + IMM land at LDS address lds + LDSOFF + 16 i (or 4 i).  (The
// instruction's offset applies to the LDS address as well, so M0 gets
// LDSOFF - IMM.)
// Non-temporal (nt): each byte is read once per call, and streaming past the
// caches is markedly faster than allocating the lines.  Written as asm so
// that the address stays in the scalar-base form (64-bit row pointer in
// SGPRs, the lane's constant 32-bit offset in a VGPR: no vector address
// arithmetic) and the LDS address is formed in M0 from one base (no scalar
// register per stage and load); the s_nop is the wait the M0 write needs
// before an LDS-DMA load.  The loads write no registers; the kernel waits
// for them with explicit vmcnt waits.
template <int IMM, int LDSOFF>
__device__ __forceinline__ void dma16(const void* sbase, uint32_t voff, uint32_t lds) {
  static_assert(IMM >= 0 && LDSOFF >= IMM && IMM < 4096, "offsets");
  asm volatile(
      "s_add_u32 m0, %0, %4\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, %2 offset:%3 nt"
      :
      : "s"(lds), "v"(voff), "s"(sbase), "i"(IMM), "i"(LDSOFF - IMM)
      : "memory", "m0", "scc");
}
template <int LDSOFF>
__device__ __forceinline__ void dma4(const void* sbase, uint32_t voff, uint32_t lds) {
  asm volatile("s_add_u32 m0, %0, %3\n\ts_nop 0\n\tglobal_load_lds_dword %1, %2 nt"
               :
               : "s"(lds), "v"(voff), "s"(sbase), "i"(LDSOFF)
               : "memory", "m0", "scc");
}

// Wait until at most N vector-memory operations of this wave are in flight.
template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

// Eight codes of one K word (nibble n = dim n of the word) as an MFMA
// operand, k-slots (n0, n4, n1, n5, n2, n6, n3, n7); odd nibbles carry 16x.
__device__ __forceinline__ h8 k_operand(uint32_t w) {
  const uint32_t w8 = w >> 8;
  const u32x4 r = {w & 0x000F000Fu, w & 0x00F000F0u, w8 & 0x000F000Fu, w8 & 0x00F000F0u};
  return __builtin_bit_cast(h8, r);
}
// Dim K of a 4-dim chunk at eight positions from four position-pair V words
// (word r: positions 2r and 2r+1) as 16 code * 2^-24, subnormal fp16
// operands: every nibble is moved to bits 4..7 of its half (the matrix cores
// sum products of the smallest subnormals, code * 2^-24, with a bias of a few
// fp32 ulps, which the centring's cancellation would amplify); k-slots in
// position order.  m holds the mask in a register (see opaque).
template <int K>
__device__ __forceinline__ h8 v_operand(uint32_t w0, uint32_t w1, uint32_t w2, uint32_t w3,
                                        uint32_t m) {
  auto f = [m](uint32_t w) {
    if constexpr (K == 0) return (w << 4) & m;
    else if constexpr (K == 1) return w & m;
    else if constexpr (K == 2) return (w >> 4) & m;
    else return (w >> 8) & m;
  };
  const u32x4 r = {f(w0), f(w1), f(w2), f(w3)};
  return __builtin_bit_cast(h8, r);
}
// A value the compiler cannot see through (no instruction is emitted): a
// constant passed through it stays in a register instead of being folded
// into a literal operand.
__device__ __forceinline__ uint32_t opaque(uint32_t v) {
  asm volatile("" : "+v"(v));
  return v;
}
// f(integral_constant<int, 0>), ..., f(integral_constant<int, N - 1>), in order.
template <int N, int I = 0, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (I < N) {
    f(std::integral_constant<int, I>{});
    static_for<N, I + 1>(f);
  }
}

__device__ __forceinline__ f32x4 mfma(h8 a, h8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
}

// All LDS reads of one staged row, waited for once (asm: the compiler would
// otherwise order every LDS read after all outstanding LDS-DMA loads).  Per
// lane: the K codes of its position in both 16-position tiles, the (scale,
// bias) words of its eight positions for K and for V, and the V words of its
// four position pairs for each of its 4-dim chunks.  OFF is the stage
// offset; kma and vma address the K and V meta words of the lane's columns.
template <int OFF>
__device__ __forceinline__ void read_row_d128(uint32_t ka, uint32_t kma, uint32_t vma,
                                              uint32_t va0, uint32_t va1, uint4& k0, uint4& k1,
                                              uint4& km0, uint4& km1, uint4& vm0, uint4& vm1,
                                              uint32_t (&v)[2][4]) {
  asm volatile(
      "ds_read_b128 %0, %14 offset:%19\n\t"
      "ds_read_b128 %1, %14 offset:%22\n\t"
      "ds_read_b128 %2, %15 offset:%19\n\t"
      "ds_read_b128 %3, %15 offset:%20\n\t"
      "ds_read_b128 %4, %16 offset:%19\n\t"
      "ds_read_b128 %5, %16 offset:%20\n\t"
      "ds_read_b32 %6, %17 offset:%19\n\t"
      "ds_read_b32 %7, %17 offset:%21\n\t"
      "ds_read_b32 %8, %17 offset:%22\n\t"
      "ds_read_b32 %9, %17 offset:%23\n\t"
      "ds_read_b32 %10, %18 offset:%19\n\t"
      "ds_read_b32 %11, %18 offset:%21\n\t"
      "ds_read_b32 %12, %18 offset:%22\n\t"
      "ds_read_b32 %13, %18 offset:%23\n\t"
      "s_waitcnt lgkmcnt(0)"
      : "=&v"(k0), "=&v"(k1), "=&v"(km0), "=&v"(km1), "=&v"(vm0), "=&v"(vm1), "=&v"(v[0][0]),
        "=&v"(v[0][1]), "=&v"(v[0][2]), "=&v"(v[0][3]), "=&v"(v[1][0]), "=&v"(v[1][1]),
        "=&v"(v[1][2]), "=&v"(v[1][3])
      : "v"(ka), "v"(kma), "v"(vma), "v"(va0), "v"(va1), "i"(OFF), "i"(OFF + 16),
        "i"(OFF + 128), "i"(OFF + 256), "i"(OFF + 384)
      : "memory");
}
// head_dim 64: 8-byte K quarters; K and V meta at separate bases.
template <int OFF>
__device__ __forceinline__ void read_row_d64(uint32_t ka, uint32_t kma, uint32_t vma, uint32_t va,
                                             uint2& k0, uint2& k1, uint4& km0, uint4& km1,
                                             uint4& vm0, uint4& vm1, uint32_t (&v)[1][4]) {
  asm volatile(
      "ds_read_b64 %0, %10 offset:%14\n\t"
      "ds_read_b64 %1, %10 offset:%17\n\t"
      "ds_read_b128 %2, %11 offset:%14\n\t"
      "ds_read_b128 %3, %11 offset:%15\n\t"
      "ds_read_b128 %4, %12 offset:%14\n\t"
      "ds_read_b128 %5, %12 offset:%15\n\t"
      "ds_read_b32 %6, %13 offset:%14\n\t"
      "ds_read_b32 %7, %13 offset:%16\n\t"
      "ds_read_b32 %8, %13 offset:%17\n\t"
      "ds_read_b32 %9, %13 offset:%18\n\t"
      "s_waitcnt lgkmcnt(0)"
      : "=&v"(k0), "=&v"(k1), "=&v"(km0), "=&v"(km1), "=&v"(vm0), "=&v"(vm1), "=&v"(v[0][0]),
        "=&v"(v[0][1]), "=&v"(v[0][2]), "=&v"(v[0][3])
      : "v"(ka), "v"(kma), "v"(vma), "v"(va), "i"(OFF), "i"(OFF + 16), "i"(OFF + 64),
        "i"(OFF + 128), "i"(OFF + 192)
      : "memory");
}
// head_dim 256: two halves of 128 dims (GOFF: meta offset of the second
// half's groups); three waits per row.
template <int OFF, int GOFF>
__device__ __forceinline__ void read_row_d256(uint32_t ka, uint32_t kma, uint32_t vma,
                                              uint32_t va, uint4 (&k)[2][2], uint4 (&km)[2][2],
                                              uint4 (&vm)[2][2], uint32_t (&v)[4][4]) {
  asm volatile(
      "ds_read_b128 %0, %12 offset:%15\n\t"
      "ds_read_b128 %1, %12 offset:%16\n\t"
      "ds_read_b128 %2, %12 offset:%17\n\t"
      "ds_read_b128 %3, %12 offset:%18\n\t"
      "ds_read_b128 %4, %13 offset:%15\n\t"
      "ds_read_b128 %5, %13 offset:%19\n\t"
      "ds_read_b128 %6, %13 offset:%20\n\t"
      "ds_read_b128 %7, %13 offset:%21\n\t"
      "ds_read_b128 %8, %14 offset:%15\n\t"
      "ds_read_b128 %9, %14 offset:%19\n\t"
      "ds_read_b128 %10, %14 offset:%20\n\t"
      "ds_read_b128 %11, %14 offset:%21\n\t"
      "s_waitcnt lgkmcnt(0)"
      : "=&v"(k[0][0]), "=&v"(k[1][0]), "=&v"(k[0][1]), "=&v"(k[1][1]), "=&v"(km[0][0]),
        "=&v"(km[0][1]), "=&v"(km[1][0]), "=&v"(km[1][1]), "=&v"(vm[0][0]), "=&v"(vm[0][1]),
        "=&v"(vm[1][0]), "=&v"(vm[1][1])
      : "v"(ka), "v"(kma), "v"(vma), "i"(OFF), "i"(OFF + 64), "i"(OFF + 512), "i"(OFF + 576),
        "i"(OFF + 16), "i"(OFF + GOFF), "i"(OFF + GOFF + 16)
      : "memory");
#pragma unroll
  for (int c2 = 0; c2 < 2; ++c2) {
    asm volatile(
        "ds_read_b32 %0, %8 offset:%9\n\t"
        "ds_read_b32 %1, %8 offset:%10\n\t"
        "ds_read_b32 %2, %8 offset:%11\n\t"
        "ds_read_b32 %3, %8 offset:%12\n\t"
        "ds_read_b32 %4, %8 offset:%13\n\t"
        "ds_read_b32 %5, %8 offset:%14\n\t"
        "ds_read_b32 %6, %8 offset:%15\n\t"
        "ds_read_b32 %7, %8 offset:%16\n\t"
        "s_waitcnt lgkmcnt(0)"
        : "=&v"(v[2 * c2][0]), "=&v"(v[2 * c2][1]), "=&v"(v[2 * c2][2]), "=&v"(v[2 * c2][3]),
          "=&v"(v[2 * c2 + 1][0]), "=&v"(v[2 * c2 + 1][1]), "=&v"(v[2 * c2 + 1][2]),
          "=&v"(v[2 * c2 + 1][3])
        : "v"(va + 128 * c2), "i"(OFF), "i"(OFF + 256), "i"(OFF + 512), "i"(OFF + 768),
          "i"(OFF + 64), "i"(OFF + 320), "i"(OFF + 576), "i"(OFF + 832)
        : "memory");
  }
}

// Page-aligned split s of n_pages pages into S parts (remainder first).
__device__ __forceinline__ void split_range(int n_pages, int S, int s, int& pb, int& pe) {
  const int base = n_pages / S, rem = n_pages % S;
  pb = s * base + min(s, rem);
  pe = pb + base + (s < rem ? 1 : 0);
}

// Coherent (sc1: device-scope) buffer loads of split records; the resource
// covers one head's records, so every access is bounds-checked by the
// hardware as well.
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
constexpr int kCpolSc1 = 16;
__device__ __forceinline__ __amdgpu_buffer_rsrc_t records_rsrc(const float* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(base), (short)0, (int)bytes,
                                           0x00020000);
}

// Row of (request b, head slot vh) in q and out.  With sq query tokens per
// request (the short verifier) the kernel's Hq heads are Hq / sq query heads
// times sq tokens: vh = head * sq + token, stored token-major
// ([B][sq][Hq / sq][D]); sq = 1 is single-query decode ([B][Hq][D]).
__device__ __forceinline__ size_t qrow(int b, int vh, int Hq, int sq) {
  return ((size_t)b * sq + vh % sq) * (Hq / sq) + vh / sq;
}

// Log-sum-exp combine of the split records of heads h0 .. h0+nh-1 (nh <= 4)
// of request b: M = max m_s, w_s = l_s 2^(m_s - M), o = sum w_s o_s / sum w_s.
// WPH waves per head: wave w combines dims [D/WPH (w % WPH), +D/WPH) of head
// w / WPH.  Lane (c, k) holds 4 of those dims (chunk c) and the splits
// s = k, k + KP, ... (KP = lanes per chunk), fetched KCH at a time with
// coherent loads and folded into a running maximum; the KP parts meet by
// shuffles.  Records: [max_splits][D + 4] fp32 per head (o/l in 0..D-1, m at
// D, l at D+1).
template <int D, int WPH, int NW>
__device__ void combine_splits(const float* ws, __half* out, int b, int Hq, int sq, int h0,
                               int nh, int max_splits, int S) {
  constexpr int DW = D / WPH;     // dims per wave
  constexpr int CPL = DW / 4;     // float4 chunks per wave
  constexpr int KP = 64 / CPL;    // lanes per chunk (split parts)
  constexpr int KCH = (32 / KP) < 16 ? (32 / KP > 0 ? 32 / KP : 1) : 16;  // splits per lane per round
  static_assert(KP >= 1 && 64 % CPL == 0, "");
  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // scalar: the records' resource too
  const int d0 = DW * (w % WPH);
  const int c = lane % CPL, k = lane / CPL;
  // wave w combines heads w / WPH, w / WPH + NW / WPH, ...
  for (int h = w / WPH; h < nh; h += NW / WPH) {
    const float* recs = ws + ((size_t)b * Hq + h0 + h) * max_splits * (D + 4);
    const __amdgpu_buffer_rsrc_t rs = records_rsrc(recs, (uint32_t)S * (D + 4) * 4);
    float m_run = -INFINITY, den = 0.0f;
    float num[4] = {0.0f, 0.0f, 0.0f, 0.0f};
    for (int s0 = k; s0 < S; s0 += KP * KCH) {
      f32x4 o[KCH];
      f32x2 ml[KCH];
#pragma unroll
      for (int i = 0; i < KCH; ++i) {
        const int s = min(s0 + KP * i, S - 1);  // past the end: a valid record, weight 0
        o[i] = __builtin_amdgcn_raw_buffer_load_b128(rs, (s * (D + 4) + d0 + 4 * c) * 4, 0, kCpolSc1);
        ml[i] = __builtin_amdgcn_raw_buffer_load_b64(rs, (s * (D + 4) + D) * 4, 0, kCpolSc1);
      }
      // (selects, not branches: the records' validity is per lane)
      float mv[KCH];
      float mx = m_run;
#pragma unroll
      for (int i = 0; i < KCH; ++i) {
        const bool on = (s0 + KP * i < S) & (ml[i].y > 0.0f);
        mv[i] = on ? ml[i].x : -INFINITY;
        mx = fmaxf(mx, mv[i]);
      }
      const float f = (m_run == -INFINITY) ? 0.0f : __builtin_amdgcn_exp2f(m_run - mx);
      den *= f;
#pragma unroll
      for (int e = 0; e < 4; ++e) num[e] *= f;
#pragma unroll
      for (int i = 0; i < KCH; ++i) {
        const float wt = (mv[i] == -INFINITY) ? 0.0f : ml[i].y * __builtin_amdgcn_exp2f(mv[i] - mx);
        den += wt;
        num[0] = fmaf(wt, o[i].x, num[0]);
        num[1] = fmaf(wt, o[i].y, num[1]);
        num[2] = fmaf(wt, o[i].z, num[2]);
        num[3] = fmaf(wt, o[i].w, num[3]);
      }
      m_run = mx;
    }
    // merge the KP parts of each chunk (lanes c, c + CPL, ...)
#pragma unroll
    for (int off = CPL; off < 64; off <<= 1) {
      const float mo = __shfl_xor(m_run, off);
      const float M = fmaxf(m_run, mo);
      const float fa = (m_run == -INFINITY) ? 0.0f : __builtin_amdgcn_exp2f(m_run - M);
      const float fb = (mo == -INFINITY) ? 0.0f : __builtin_amdgcn_exp2f(mo - M);
      den = den * fa + __shfl_xor(den, off) * fb;
#pragma unroll
      for (int e = 0; e < 4; ++e) num[e] = num[e] * fa + __shfl_xor(num[e], off) * fb;
      m_run = M;
    }
    if (k == 0) {
      const float r = den > 0.0f ? 1.0f / den : 0.0f;
      __half2* dst = reinterpret_cast<__half2*>(out + qrow(b, h0 + h, Hq, sq) * D + d0 + 4 * c);
      dst[0] = __floats2half2_rn(num[0] * r, num[1] * r);
      dst[1] = __floats2half2_rn(num[2] * r, num[3] * r);
    }
  }
}

// Decode kernel.  Block = 8 (d <= 128) or 4 waves = one split of one
// (request, KV head, head chunk).  A chunk is CS column sets of H head slots
// (H = head_slots(): 8 for 64- and 128-dim groups at d <= 128, 4 for 32-dim
// groups or d = 256); the sets share every row's K and V operands and keep
// their own softmax state and accumulators.  Lane (m, q) =
// (lane % 16, lane / 16) feeds row m
// and k-quarter q of the MFMA operands and receives column m, rows 4q..4q+3
// of the 16x16 results.
//   scores: tile t (0, 1) row m = position 8 (m / 4) + 4 t + m % 4 of the row,
//           A = the lane's K quarter (dims q D/4 .. of each 128-dim half),
//           B = Q' of the set (column h + H s: head h, dims of the scale
//           group slot s stands for only);
//           result lane (col, q), element i = position 8 q + 4 t + i;
//   values: tile (c, k) row m = dim 4 (16 c + m) + k, A = positions 8 q .. 8 q
//           + 7 (the lane's four position pairs) of that dim, B = W of the
//           same positions (exactly the lane's eight score positions), so the
//           scores never leave their lanes.
// Progress: every wave runs the same number of ring cycles (its last ones
// without rows) and the block's waves meet at a barrier after each cycle.
//
// APPEND (the fused decode step): in the block of each request's last split,
// the wave that streams the row holding position seq_lens[b] - 1 quantizes
// the request's new K/V row (fp16 [B][Hkv][d], one per request) for its KV
// head while its first page loads are in flight, stores it to the pool
// without waiting, and writes the same bytes into its LDS stage once that
// row's loads have landed (they may still see the slot's previous bytes);
// no other block reads that page.
template <int D, int G, bool APPEND, int CS>
__global__ __launch_bounds__(kMaxThreads) void decode_kernel(
    uint8_t* __restrict__ k_codes, uint32_t* __restrict__ k_meta,
    uint8_t* __restrict__ v_codes, uint32_t* __restrict__ v_meta,
    const uint4* __restrict__ k_new, const uint4* __restrict__ v_new,
    const __half* __restrict__ q, const int32_t* __restrict__ block_tables,
    const int32_t* __restrict__ seq_lens, float* __restrict__ ws, uint32_t* __restrict__ tickets,
    __half* __restrict__ out, int Hq, int sq, int Hkv, int P, int NP, int max_pages,
    int max_splits, int split_cap, int n_hchunks, float scale_log2) {
  constexpr int kWaves = waves_for<D>();
  constexpr int kThreads = 64 * kWaves;
  constexpr int NG = D / G;                // scale groups per head
  constexpr int HD = D < 128 ? D : 128;    // dims per half
  constexpr int NHALF = D / HD;            // halves: separate score accumulators
  constexpr int DQ = HD / 4;               // dims of a k-quarter per half
  constexpr int WQ = DQ / 8;               // its code words: MFMA steps per half and tile
  constexpr int NC = D / 64;               // 16-chunk blocks of 4 dims (value tiles: 4 NC)
  constexpr int KB = kRowPos * D / 2;      // K (and V) code bytes per row
  constexpr int K_DMAS = KB / 1024;        // 16-byte LDS-DMA loads per row, K (and V)
  constexpr int META_WORDS = kRowPos * NG;
  constexpr int META_DMAS = (META_WORDS + 63) / 64;
  constexpr int kMetaBytes = 256 * META_DMAS;  // K or V (scale, bias) words per row
  constexpr int kStageBytes = 2 * KB + 2 * kMetaBytes;
  constexpr int DMAS_PER_ROW = 2 * K_DMAS + 2 * META_DMAS;
  constexpr int kFit = (kRingBudget - 16) / (kWaves * kStageBytes);
  constexpr int kStages = kFit < kMaxStages ? kFit : kMaxStages;
  static_assert(kStages >= 2, "ring depth");
  constexpr int kHeadSlots = head_slots<D, G>();  // heads per column set
  constexpr int NS = 16 / kHeadSlots;      // column slots per head
  constexpr int kChunk = kHeadSlots * CS;  // heads per block: CS column sets
  static_assert(kChunk <= kWaves ? kWaves % kChunk == 0 : kChunk % kWaves == 0,
                "whole waves per head, or whole heads per wave, in the combine");
  constexpr bool kSwz = (D == 128);
  static_assert(DMAS_PER_ROW * (kStages - 1) < 64, "vmcnt range");
  static_assert(kChunk * D + 2 * kChunk <= kStages * kStageBytes / 4, "merge fits a ring");

  __shared__ __attribute__((aligned(16))) uint8_t smem[kWaves][kStages][kStageBytes];
  __shared__ uint32_t s_ticket;

  // Block -> (split, KV head, head chunk).  One head chunk: x = split,
  // y = KV head.  Several chunks read the same pages, so their blocks are
  // placed on one XCD (blocks are dealt to the XCDs in turn by linear ID):
  // x = group * (kXcds * n_hchunks) + hc * kXcds + lane, where slot
  // group * kXcds + lane is (split, KV head); the chunks of a slot then share
  // that XCD's L2 while they stream the same rows.
  int split, kv, hc;
  if (n_hchunks == 1) {
    split = blockIdx.x;
    kv = blockIdx.y;
    hc = 0;
  } else {
    const int per = kXcds * n_hchunks;
    const int g = blockIdx.x / per, r = blockIdx.x % per;
    const int slot = g * kXcds + r % kXcds;
    hc = r / kXcds;
    split = slot % split_cap;
    kv = slot / split_cap;
    if (kv >= Hkv) return;  // padding of the last group
  }
  const int b = blockIdx.z;
  const int gq = Hq / Hkv;
  const int h0 = kv * gq + hc * kChunk;
  const int nh = min(kChunk, gq - hc * kChunk);
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // wave-uniform (scalar)

  const int l16 = lane & 15, q4 = lane >> 4;
  const int hs = l16 % kHeadSlots, gs = l16 / kHeadSlots;  // accumulator column: head, slot
  // column set cs holds heads cs kHeadSlots + hs of the chunk
  bool head_on[CS];
  int hsel[CS];  // the head whose query this lane's column reads (a valid one)
#pragma unroll
  for (int cs = 0; cs < CS; ++cs) {
    head_on[cs] = cs * kHeadSlots + hs < nh;
    hsel[cs] = min(cs * kHeadSlots + hs, nh - 1);
  }

  // Loads issued together, before anything waits for the request's length:
  // the query words of head hs over the dims of quarter q4 (the lane's
  // k-slots), the page IDs of this split's range as it is when the request
  // fills its table (the common case; read again below otherwise), and, in
  // the fused step, the new row's fp16 values (lanes 0 .. D/8 - 1: K dims
  // 8 lane ..; lanes D/8 .. D/4 - 1: V) in the block that would hold it.
  uint4 qraw[CS][NHALF][WQ];
#pragma unroll
  for (int cs = 0; cs < CS; ++cs) {
    const uint4* src = reinterpret_cast<const uint4*>(
        q + qrow(b, h0 + hsel[cs], Hq, sq) * D + DQ * q4);
#pragma unroll
    for (int e = 0; e < NHALF; ++e)
#pragma unroll
      for (int kb = 0; kb < WQ; ++kb) qraw[cs][e][kb] = src[(HD / 8) * e + kb];
  }
  const int S_full = min(split_cap, max_pages);
  int pb_full, pe_full;
  split_range(max_pages, S_full, split, pb_full, pe_full);
  const int pg_full = (split < S_full && lane < pe_full - pb_full)
                          ? block_tables[(size_t)b * max_pages + pb_full + lane]
                          : -1;
  const int app_kind = lane / (D / 8), app_c8 = lane % (D / 8);
  // (every lane loads, lanes D/4 .. again from K or V, so that the branch
  // stays block-uniform and the value is not needed before it is used)
  const uint4* app_src = ((app_kind & 1) ? v_new : k_new) + ((size_t)b * Hkv + kv) * (D / 8) + app_c8;
  uint4 app_x;
  if constexpr (APPEND) {
    if (split == S_full - 1) app_x = *app_src;
  }

  const int L = min(seq_lens[b], max_pages * P);
  if (L <= 0) {  // an empty request: all-zero output rows, written by split 0
    if (split == 0)
      for (int i = tid; i < nh * D; i += kThreads)
        out[qrow(b, h0 + i / D, Hq, sq) * D + i % D] = __float2half(0.0f);
    return;
  }
  const int n_pages = (L + P - 1) / P;
  const int S = min(split_cap, n_pages);  // split_cap <= max_splits (the record stride)
  if (split >= S) return;
  int pb, pe;
  split_range(n_pages, S, split, pb, pe);
  const int t_end = min(pe * P, L);
  // causal limits of the verifier: token k of sq sees positions < L - sq + 1
  // + k (its own and those before it); rows below t_full need no mask
  const int t_full = min(t_end, L - sq + 1);
  int t_lim[CS];
#pragma unroll
  for (int cs = 0; cs < CS; ++cs) t_lim[cs] = min(t_end, L - sq + 1 + (h0 + hsel[cs]) % sq);
  const int rows_per_page = P / kRowPos;

  // this wave's rows: the split's rows in page order, wave, wave + kWaves, ...
  const int n_split_pages = pe - pb;
  const int split_rows = n_split_pages * rows_per_page;
  const int my_rows = (split_rows > wave) ? (split_rows - wave + kWaves - 1) / kWaves : 0;
  const size_t head_codes = (size_t)P * (D / 2);
  const size_t page_codes = (size_t)Hkv * head_codes;
  uint8_t* ring = smem[wave][0];
  const uint32_t ring_lds = (uint32_t)(uintptr_t)ring;

  // The split's page IDs, 64 per vector register (lane k holds page pb + k of
  // the group), read with v_readlane when the issue cursor enters a page.
  auto load_group = [&](int grp) {
    const int k = 64 * grp + lane;
    return (k < n_split_pages) ? block_tables[(size_t)b * max_pages + pb + k] : -1;
  };
  const bool full_table = n_pages == max_pages;  // then pb, pe are pb_full, pe_full
  int pg_grp = full_table ? pg_full : load_group(0);
  int cur_grp = 0;

  // The fused step's new row, at position seq_lens[b] - 1 = L - 1, lies in
  // the last row of the last split.  The wave that streams that row
  // quantizes it (below, once its first page loads are in flight): it
  // stores the codes and (scale, bias) words to the pool, and writes the
  // same bytes into its LDS stage after the row's page loads have landed,
  // since those loads may still see the slot's previous bytes.  Nothing
  // waits for the stores.
  int app_pos = -1;  // >= 0: this wave appends the row at that position
  if constexpr (APPEND) {
    const int pos = seq_lens[b] - 1;
    if (split == S - 1 && pos < max_pages * P && ((pos - pb * P) / kRowPos) % kWaves == wave) {
      app_pos = pos;
      if (!full_table) app_x = *app_src;
    }
  }

  // Per-lane parts of the load addresses (the row parts are scalar).  A DMA
  // lane stores 16 bytes at 16 * lane, so the chunk a lane fetches decides
  // the LDS layout.  d = 128: K quarter q of position p sits in slot
  // q ^ f(p) of the position (f: bits 1 and 3 of p), V chunk u of pair s in
  // slot u ^ 4 ((s / 4) & 1) of the pair, so the lanes of one read
  // instruction spread over the banks.
  uint32_t k_off, v_off;
  if constexpr (kSwz) {
    const int p = lane >> 2, j = lane & 3;
    const int f = ((p >> 1) & 1) | (((p >> 3) & 1) << 1);
    k_off = 64u * p + 16u * (j ^ f);
    const int s = lane >> 3, u4 = lane & 7;
    v_off = (uint32_t)D * s + 16u * (u4 ^ (4 * ((s >> 2) & 1)));
  } else {
    k_off = v_off = 16u * lane;
  }
  uint32_t meta_off[META_DMAS];  // LDS word w = (group w / 32, position w % 32)
#pragma unroll
  for (int i = 0; i < META_DMAS; ++i) {
    const int w = 64 * i + lane;
    const int wi = (w < META_WORDS) ? w : 0;
    meta_off[i] = 4u * (uint32_t)((wi % kRowPos) * NG + wi / kRowPos);
  }

  // Issue cursor: the next row to load (page ipk of the split, row irr of the
  // page) and the scalar addresses of that row.
  int ipk = wave / rows_per_page, irr = wave % rows_per_page;
  const uint8_t* ik = k_codes;
  const uint8_t* iv = v_codes;
  const uint8_t* ikm = reinterpret_cast<const uint8_t*>(k_meta);
  const uint8_t* ivm = reinterpret_cast<const uint8_t*>(v_meta);
  bool iok = false;
  auto enter_page = [&]() {
    if ((ipk >> 6) != cur_grp) {  // more than 64 pages per split: next 64 IDs
      cur_grp = ipk >> 6;
      pg_grp = load_group(cur_grp);
      wait_vm<0>();  // here, so that the common path carries no pending load
    }
    int page = __builtin_amdgcn_readlane(pg_grp, ipk & 63);
    iok = (unsigned)page < (unsigned)NP;
    if (!iok) page = 0;  // never read past the pool; the positions are masked
    const size_t run = (size_t)page * Hkv + kv;
    ik = k_codes + run * head_codes + (size_t)irr * KB;
    iv = v_codes + run * head_codes + (size_t)irr * KB;
    const size_t mo = (run * P + (size_t)irr * kRowPos) * NG * 4;
    ikm = reinterpret_cast<const uint8_t*>(k_meta) + mo;
    ivm = reinterpret_cast<const uint8_t*>(v_meta) + mo;
  };
  bool stage_ok[kStages];
  // Loads of the next row into stage ST; past the wave's last row, loads of
  // one 16-byte run by every lane (same count, negligible traffic) keep the
  // number of loads in flight per row constant.
  auto issue = [&](auto st_c, bool real) {
    constexpr int ST = decltype(st_c)::value;
    uint8_t* st = ring + ST * kStageBytes;
    constexpr int SO = ST * kStageBytes;  // the stage's offset in the ring
    if (real) {
      static_for<K_DMAS>([&](auto c_c) {
        constexpr int C = decltype(c_c)::value;
        dma16<1024 * C, SO + 1024 * C>(ik, k_off, ring_lds);
      });
      static_for<K_DMAS>([&](auto c_c) {
        constexpr int C = decltype(c_c)::value;
        dma16<1024 * C, SO + KB + 1024 * C>(iv, v_off, ring_lds);
      });
      static_for<META_DMAS>([&](auto i_c) {
        constexpr int I = decltype(i_c)::value;
        dma4<SO + 2 * KB + 256 * I>(ikm, meta_off[I], ring_lds);
        dma4<SO + 2 * KB + kMetaBytes + 256 * I>(ivm, meta_off[I], ring_lds);
      });
      stage_ok[ST] = iok;
      // advance the cursor by kWaves rows
      irr += kWaves;
      if (irr < rows_per_page) {
        ik += kWaves * KB;
        iv += kWaves * KB;
        ikm += kWaves * kRowPos * NG * 4;
        ivm += kWaves * kRowPos * NG * 4;
      } else {
        do {
          irr -= rows_per_page;
          ++ipk;
        } while (irr >= rows_per_page);
        if (ipk < n_split_pages) enter_page();
      }
    } else {  // past the last row: the first bytes of the pool, never used
      static_for<2 * K_DMAS>([&](auto c_c) {
        dma16<0, SO + 1024 * decltype(c_c)::value>(k_codes, 0u, ring_lds);
      });
      static_for<2 * META_DMAS>([&](auto i_c) {
        dma4<SO + 2 * KB + 256 * decltype(i_c)::value>(k_meta, 0u, ring_lds);
      });
      stage_ok[ST] = false;
    }
  };
  wait_vm<0>();  // page IDs and query words (issued together) have arrived
  if (my_rows > 0) enter_page();
  // All stages are in flight while a row is computed: a row's stage is read
  // into registers first and then refilled with the row kStages ahead.
  if (my_rows > 0) {
    static_for<kStages>([&](auto st_c) { issue(st_c, decltype(st_c)::value < my_rows); });
  }

  // ---- the fused step's row: quantized by the whole wave (the first page
  // loads are in flight meanwhile), then stored to the pool
  uint32_t app_packed = 0, app_meta = 0;
  if constexpr (APPEND) {
    if (app_pos >= 0) {
      app_packed = jfkv::quantize8(app_x, G / 8, app_meta);
      const int pidx = app_pos / P - pb;  // wave-uniform
      const int page = ((pidx >> 6) == cur_grp)
                           ? __builtin_amdgcn_readlane(pg_grp, pidx & 63)
                           : block_tables[(size_t)b * max_pages + app_pos / P];
      if (app_kind < 2 && (unsigned)page < (unsigned)NP)
        jfkv::store_codes8(app_kind ? v_codes : k_codes, app_kind ? v_meta : k_meta,
                           app_kind != 0, (int64_t)page * Hkv + kv, P, D, G, app_pos % P, app_c8,
                           G / 8, app_packed, app_meta);
    }
  }

  // ---- Q' operands.  Score column hs + kHeadSlots gs holds head hs
  // restricted to the dims of scale group gs % NGH of each half (columns with
  // equal group are copies), so each column's sum has one scale; k-slots (n0,
  // n4, n1, n5, n2, n6, n3, n7) of each code word, odd nibbles' dims divided
  // by 16.  qs: the group's query sum (times 2^-24, the code scale), its bias
  // factor.  The value column of the same slot carries the same group.
  constexpr int NGH = HD / G;            // scale groups per half
  static_assert(NS % NGH == 0, "every group of a half has a column slot");
  const int gcol = gs % NGH;             // group (within a half) of the column
  // a negative softmax scale negates the query (exact) and leaves |scale|
  const uint32_t qneg = scale_log2 < 0.0f ? 0x80008000u : 0u;
  h8 qB[CS][NHALF][WQ];
  float qs[CS][NHALF];
#pragma unroll
  for (int cs = 0; cs < CS; ++cs)
#pragma unroll
  for (int e = 0; e < NHALF; ++e) {
    const bool q_on = head_on[cs] && (DQ * q4) / G == gcol;
    float s = 0.0f;
#pragma unroll
    for (int kb = 0; kb < WQ; ++kb) {
      const uint4 u = qraw[cs][e][kb];
      const uint32_t wq[4] = {u.x ^ qneg, u.y ^ qneg, u.z ^ qneg, u.w ^ qneg};
      _Float16 x[8];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        x[2 * i] = as_h2(wq[i]).x;
        x[2 * i + 1] = as_h2(wq[i]).y;
      }
#pragma unroll
      for (int i = 0; i < 8; ++i) s += (float)x[i];
      const _Float16 sixteenth = (_Float16)0.0625f;
      h8 o = {x[0], x[4], x[1] * sixteenth, x[5] * sixteenth,
              x[2], x[6], x[3] * sixteenth, x[7] * sixteenth};
      if (!q_on) o = h8{};
      qB[cs][e][kb] = o;
    }
    // the group's query sum: quarter sums of the four lanes l16 + 16 k
    const float sq[4] = {s, __shfl_xor(s, 16), __shfl_xor(s, 32), __shfl_xor(s, 48)};
    float g = 0.0f;
#pragma unroll
    for (int k = 0; k < 4; ++k)
      if ((DQ * (q4 ^ k)) / G == gcol) g += sq[k];
    qs[cs][e] = head_on[cs] ? g * (1.0f / 16777216.0f) : 0.0f;
  }
  // 2^24 (the code scale) times |scale| in log2 units; a positive floor keeps
  // masked (-inf) scores at -inf when the scale is 0
  const float kfold = 16777216.0f * fmaxf(fabsf(scale_log2), 1e-30f);

  f32x4 acc_o[CS][NC][4];
  float m_run[CS], thr[CS], l_run[CS];
  // The value groups' sums of p * bias and of p * scale - W.  d <= 128: both
  // from matrix-core products into acc_bs, whose A operand rows are group
  // g's bias (row g H), its scale (row g H + 1, where a second product with
  // A = -1 subtracts W in the same accumulator) and zeros elsewhere (H head
  // slots: lanes g H .. hold group g's (scale, bias) words); d = 256: per-lane
  // dot products.
  constexpr bool kSumMfma = NHALF == 1;
  f32x4 acc_bs[CS];
  float bacc[CS][NHALF], sacc8[CS][NHALF];
#pragma unroll
  for (int cs = 0; cs < CS; ++cs) {
#pragma unroll
    for (int c = 0; c < NC; ++c)
#pragma unroll
      for (int k = 0; k < 4; ++k) acc_o[cs][c][k] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
    m_run[cs] = thr[cs] = kMinit;
    l_run[cs] = 0.0f;
    acc_bs[cs] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int e = 0; e < NHALF; ++e) bacc[cs][e] = sacc8[cs][e] = 0.0f;
  }
  const int s_grp = l16 / kHeadSlots, s_row = l16 % kHeadSlots;  // the lane's sum row role
  const bool s_bias = s_grp < NGH && s_row == 0, s_scale = s_grp < NGH && s_row == 1;
  const uint32_t s_sel = s_bias ? 0x07060302u : s_scale ? 0x05040100u : 0x0C0C0C0Cu;
  const _Float16 s_neg = s_scale ? (_Float16)-1.0f : (_Float16)0.0f;
  const h8 s_aw = {s_neg, s_neg, s_neg, s_neg, s_neg, s_neg, s_neg, s_neg};

  // LDS read bases (stage 0)
  const int p0 = 8 * (l16 >> 2) + (l16 & 3);  // tile-0 position of row m = l16
  uint32_t ka, kma, vma, va[NC];
  if constexpr (D == 128) {
    const int f = ((p0 >> 1) & 1) | (((p0 >> 3) & 1) << 1);
    ka = ring_lds + 64 * p0 + 16 * (q4 ^ f);
  } else if constexpr (D == 256) {
    ka = ring_lds + 128 * p0 + 16 * q4;
  } else {
    ka = ring_lds + 32 * p0 + 8 * q4;
  }
  {
    kma = ring_lds + 2 * KB + (gcol * kRowPos + 8 * q4) * 4;  // score column's group
    vma = ring_lds + 2 * KB + kMetaBytes + (gcol * kRowPos + 8 * q4) * 4;  // (first half)
  }
#pragma unroll
  for (int c = 0; c < NC; ++c) {
    const int u4 = 4 * c + (l16 >> 2);
    va[c] = ring_lds + KB + 4 * q4 * D + 16 * (kSwz ? (u4 ^ (4 * (q4 & 1))) : u4) + 4 * (l16 & 3);
  }

  int t_row = pb * P + wave * kRowPos;  // first logical position of the row
  int issued_rows = kStages;            // rows whose loads were issued (incl. past the end)
  const h2 ones = {(_Float16)1.0f, (_Float16)1.0f};
  const uint32_t vmask = opaque(0x00F000F0u);
  const h2 mones = {(_Float16)-1.0f, (_Float16)-1.0f};
  auto row = [&](auto st_c) {
    constexpr int ST = decltype(st_c)::value;
    constexpr int OFF = ST * kStageBytes;
    // wait until only the kStages - 1 rows after this one are in flight
    wait_vm<DMAS_PER_ROW * (kStages - 1)>();
    if constexpr (APPEND) {
      // the fused step's row: its bytes in the stage, laid out as the page
      // loads place them (K quarter swizzle, V position pairs, meta
      // transposed to [group][position])
      if (app_pos >= t_row && app_pos < t_row + kRowPos) {
        const int p = app_pos - t_row;
        const uint32_t st = ring_lds + OFF;
        if (app_kind == 0) {
          const int qd = app_c8 >> 2;
          const int f = ((p >> 1) & 1) | (((p >> 3) & 1) << 1);
          const uint32_t a = st + (D / 2) * p + 16 * (kSwz ? (qd ^ f) : qd) + 4 * (app_c8 & 3);
          asm volatile("ds_write_b32 %0, %1" : : "v"(a), "v"(app_packed) : "memory");
        } else if (app_kind == 1) {
          const int sp = p >> 1, u0 = 2 * app_c8;
          const int c16 = kSwz ? ((u0 >> 2) ^ (4 * ((sp >> 2) & 1))) : (u0 >> 2);
          const uint32_t a = st + KB + D * sp + 16 * c16 + 4 * (u0 & 3) + 2 * (p & 1);
          asm volatile("ds_write_b16 %0, %1\n\tds_write_b16 %0, %2 offset:4"
                       : : "v"(a), "v"(app_packed & 0xffffu), "v"(app_packed >> 16) : "memory");
        }
        if (app_kind < 2 && (app_c8 % (G / 8)) == 0) {
          const uint32_t a = st + 2 * KB + (app_kind ? kMetaBytes : 0) +
                             4 * (((app_c8 * 8) / G) * kRowPos + p);
          asm volatile("ds_write_b32 %0, %1" : : "v"(a), "v"(app_meta) : "memory");
        }
      }
    }
    const bool pg_ok = stage_ok[ST];
    const bool full = pg_ok && t_row + kRowPos <= t_full;  // wave-uniform

    uint32_t kw[NHALF][2][WQ];   // K code words [half][tile][step]
    uint32_t kmw[NHALF][2][4];   // K (scale, bias) of positions 8 q4 + 4 t + i
    uint32_t vmw[NHALF][2][4];   // V (scale, bias), same positions
    uint32_t vw[NC][4];          // V words of pairs 4 q4 + r
    auto unpack4 = [](const uint4& u, uint32_t* w) {
      w[0] = u.x; w[1] = u.y; w[2] = u.z; w[3] = u.w;
    };
    if constexpr (D == 128) {
      uint4 k0, k1, km0, km1, vm0, vm1;
      uint32_t v[2][4];
      read_row_d128<OFF>(ka, kma, vma, va[0], va[1], k0, k1, km0, km1, vm0, vm1, v);
      unpack4(k0, kw[0][0]); unpack4(k1, kw[0][1]);
      unpack4(km0, kmw[0][0]); unpack4(km1, kmw[0][1]);
      unpack4(vm0, vmw[0][0]); unpack4(vm1, vmw[0][1]);
#pragma unroll
      for (int c = 0; c < 2; ++c)
#pragma unroll
        for (int r = 0; r < 4; ++r) vw[c][r] = v[c][r];
    } else if constexpr (D == 64) {
      uint2 k0, k1;
      uint4 km0, km1, vm0, vm1;
      uint32_t v[1][4];
      read_row_d64<OFF>(ka, kma, vma, va[0], k0, k1, km0, km1, vm0, vm1, v);
      kw[0][0][0] = k0.x; kw[0][0][1] = k0.y;
      kw[0][1][0] = k1.x; kw[0][1][1] = k1.y;
      unpack4(km0, kmw[0][0]); unpack4(km1, kmw[0][1]);
      unpack4(vm0, vmw[0][0]); unpack4(vm1, vmw[0][1]);
#pragma unroll
      for (int r = 0; r < 4; ++r) vw[0][r] = v[0][r];
    } else {
      uint4 k[2][2], km[2][2], vm[2][2];
      uint32_t v[4][4];
      read_row_d256<OFF, (128 / G) * kRowPos * 4>(ka, kma, vma, va[0], k, km, vm, v);
#pragma unroll
      for (int e = 0; e < 2; ++e)
#pragma unroll
        for (int t = 0; t < 2; ++t) {
          unpack4(k[e][t], kw[e][t]);
          unpack4(km[e][t], kmw[e][t]);
          unpack4(vm[e][t], vmw[e][t]);
        }
#pragma unroll
      for (int c = 0; c < 4; ++c)
#pragma unroll
        for (int r = 0; r < 4; ++r) vw[c][r] = v[c][r];
    }
    // the stage is in registers: refill it with the row kStages ahead
    issue(std::integral_constant<int, ST>{}, issued_rows++ < my_rows);

    // ---- scores: S^T tiles, one accumulator per half and column set (the
    // K operands are shared by the sets)
    f32x4 sacc[CS][NHALF][2];
#pragma unroll
    for (int cs = 0; cs < CS; ++cs)
#pragma unroll
      for (int e = 0; e < NHALF; ++e)
#pragma unroll
        for (int t = 0; t < 2; ++t) sacc[cs][e][t] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
#pragma unroll
    for (int kb = 0; kb < WQ; ++kb)
#pragma unroll
      for (int e = 0; e < NHALF; ++e)
#pragma unroll
        for (int t = 0; t < 2; ++t) {
          const h8 ko = k_operand(kw[e][t][kb]);
#pragma unroll
          for (int cs = 0; cs < CS; ++cs) sacc[cs][e][t] = mfma(ko, qB[cs][e][kb], sacc[cs][e][t]);
        }

    // ---- logits: fold each column's group scale and bias, sum the distinct
    // groups of the head (lanes l16 + kHeadSlots k of the 16-lane row: slots
    // gs and gs + NGH are copies, so log2(NGH) rotations suffice), scale
    // (all folds first, then the rotations: a rotation reads a value two
    // instructions after it was written at the earliest, so no wait states)
    float sc[CS][2][4];
#pragma unroll
    for (int cs = 0; cs < CS; ++cs)
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          float a = 0.0f;
#pragma unroll
          for (int e = 0; e < NHALF; ++e) a = fold_meta(kmw[e][t][i], sacc[cs][e][t][i], qs[cs][e], a);
          sc[cs][t][i] = a;  // (scaled by kfold in the exponent)
        }
#pragma unroll
    for (int cs = 0; cs < CS; ++cs)
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          if constexpr (NGH >= 2) sc[cs][t][i] = row_ror_add<kHeadSlots>(sc[cs][t][i]);
          if constexpr (NGH >= 4) sc[cs][t][i] = row_ror_add<2 * kHeadSlots>(sc[cs][t][i]);
        }
    if (__builtin_expect(!full, 0)) {
      // (an empty volatile statement keeps this a branch: the compiler would
      // otherwise compute the masks as selects on every row)
      asm volatile("" ::: "memory");
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int tp = t_row + 8 * q4 + 4 * t + i;
          // positions past the split's end or in no page: no score, and no
          // (scale, bias) words (they may hold anything)
          const bool ok = pg_ok && tp < t_end;
#pragma unroll
          for (int cs = 0; cs < CS; ++cs) sc[cs][t][i] = ok && tp < t_lim[cs] ? sc[cs][t][i] : -INFINITY;
#pragma unroll
          for (int e = 0; e < NHALF; ++e) vmw[e][t][i] = ok ? vmw[e][t][i] : 0u;
        }
    }
    h8 W[CS][NHALF];
#pragma unroll
    for (int cs = 0; cs < CS; ++cs) {
      const float mx = kfold * max8(sc[cs][0][0], sc[cs][0][1], sc[cs][0][2], sc[cs][0][3],
                                    sc[cs][1][0], sc[cs][1][1], sc[cs][1][2], sc[cs][1][3]);
      if (__builtin_amdgcn_ballot_w64(mx > thr[cs]) != 0) {
        // new running maximum of the head: lanes with equal lane % kHeadSlots
        const float M = xor_max_from(mx, kHeadSlots);
        if (M > m_run[cs]) {
          const float alpha = __builtin_amdgcn_exp2f(m_run[cs] - M);
          m_run[cs] = M;
          thr[cs] = M + kTau;
          l_run[cs] *= alpha;
          if constexpr (kSumMfma) {
            acc_bs[cs] *= alpha;
          } else {
#pragma unroll
            for (int e = 0; e < NHALF; ++e) {
              bacc[cs][e] *= alpha;
              sacc8[cs][e] *= alpha;
            }
          }
#pragma unroll
          for (int c = 0; c < NC; ++c)
#pragma unroll
            for (int k = 0; k < 4; ++k) acc_o[cs][c][k] *= alpha;
        }
      }
      // ---- p (fp16 pairs of positions 8 q4 + 2r, + 1), row sum, W = p * scale
      h2 pk[4];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int t = r >> 1, i = 2 * (r & 1);
        pk[r] = h2{(_Float16)__builtin_amdgcn_exp2f(fmaf(sc[cs][t][i], kfold, -m_run[cs])),
                   (_Float16)__builtin_amdgcn_exp2f(fmaf(sc[cs][t][i + 1], kfold, -m_run[cs]))};
        l_run[cs] = __builtin_amdgcn_fdot2(pk[r], ones, l_run[cs], false);
      }
#pragma unroll
      for (int e = 0; e < NHALF; ++e) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int t = r >> 1, i = 2 * (r & 1);
          const uint32_t a = vmw[e][t][i], c = vmw[e][t][i + 1];
          const h2 sv = as_h2(__builtin_amdgcn_perm(c, a, 0x05040100u));
          const h2 w = pk[r] * sv;
          W[cs][e][2 * r] = w.x;
          W[cs][e][2 * r + 1] = w.y;
          if constexpr (!kSumMfma) {
            const h2 bv = as_h2(__builtin_amdgcn_perm(c, a, 0x07060302u));
            bacc[cs][e] = __builtin_amdgcn_fdot2(pk[r], bv, bacc[cs][e], false);
            sacc8[cs][e] = __builtin_amdgcn_fdot2(pk[r], sv, sacc8[cs][e], false);
            sacc8[cs][e] = __builtin_amdgcn_fdot2(w, mones, sacc8[cs][e], false);
          }
        }
      }
      if constexpr (kSumMfma) {
        // rows of bias and scale (positions in the k-slot order of p), then
        // -W into the scale rows
        u32x4 am;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int t = r >> 1, i = 2 * (r & 1);
          am[r] = __builtin_amdgcn_perm(vmw[0][t][i + 1], vmw[0][t][i], s_sel);
        }
        const h8 pb = __builtin_bit_cast(h8, u32x4{__builtin_bit_cast(uint32_t, pk[0]),
                                                   __builtin_bit_cast(uint32_t, pk[1]),
                                                   __builtin_bit_cast(uint32_t, pk[2]),
                                                   __builtin_bit_cast(uint32_t, pk[3])});
        acc_bs[cs] = mfma(__builtin_bit_cast(h8, am), pb, acc_bs[cs]);
        acc_bs[cs] = mfma(s_aw, W[cs][0], acc_bs[cs]);
      }
    }
    // ---- values: O^T += V codes x W, dims 4 (16 c + m) + k (the V
    // operands are shared by the sets)
#pragma unroll
    for (int c = 0; c < NC; ++c) {
      const int e = c >> 1 < NHALF ? c >> 1 : 0;
      const h8 v0 = v_operand<0>(vw[c][0], vw[c][1], vw[c][2], vw[c][3], vmask);
      const h8 v1 = v_operand<1>(vw[c][0], vw[c][1], vw[c][2], vw[c][3], vmask);
      const h8 v2 = v_operand<2>(vw[c][0], vw[c][1], vw[c][2], vw[c][3], vmask);
      const h8 v3 = v_operand<3>(vw[c][0], vw[c][1], vw[c][2], vw[c][3], vmask);
#pragma unroll
      for (int cs = 0; cs < CS; ++cs) {
        acc_o[cs][c][0] = mfma(v0, W[cs][e], acc_o[cs][c][0]);
        acc_o[cs][c][1] = mfma(v1, W[cs][e], acc_o[cs][c][1]);
        acc_o[cs][c][2] = mfma(v2, W[cs][e], acc_o[cs][c][2]);
        acc_o[cs][c][3] = mfma(v3, W[cs][e], acc_o[cs][c][3]);
      }
    }
    t_row += kWaves * kRowPos;
  };
  // every wave runs the same number of ring cycles (block barrier per cycle)
  const int max_rows = (split_rows + kWaves - 1) / kWaves;
  for (int r0 = 0; r0 < max_rows; r0 += kStages) {
    static_for<kStages>([&](auto st_c) {
      if (r0 + decltype(st_c)::value < my_rows) row(st_c);
    });
    __syncthreads();
  }
  wait_vm<0>();  // loads issued past the last row have landed (the ring is reused)

  // ---- merge.  Each wave writes its unnormalized output (code sums times
  // the code factor plus the bias sums), its maximum and its row sum into its
  // own ring, which is idle now; after one barrier the split's threads add
  // the waves' parts, rescaled to the split's maximum.
  float* part = reinterpret_cast<float*>(ring);  // [kChunk][D]
  float* part_m = part + kChunk * D;              // [kChunk]
  float* part_l = part_m + kChunk;                // [kChunk]
  {
    const int lane_e = lane_id_volatile();
    const int me = lane_e & 15, qe = lane_e >> 4;
    const int hse = me % kHeadSlots, gse = me / kHeadSlots;
#pragma unroll
    for (int cs = 0; cs < CS; ++cs) {
      // the value groups' sums of p * (bias + 8 scale) - 8 W: the bias part
      // of the value and the centring of the codes
      float bsum[NHALF];
      if constexpr (kSumMfma) {
        // column me's group g: rows g H (element 0) and g H + 1 (element 1)
        // of acc_bs, held by lane me + 16 (g H / 4)
        const int src = me + 16 * ((((me / kHeadSlots) % NGH) * kHeadSlots) / 4);
        const float bq = __shfl(acc_bs[cs][0], src);
        const float sq8 = __shfl(acc_bs[cs][1], src);
        bsum[0] = fmaf(8.0f, sq8, bq);
      } else {
#pragma unroll
        for (int e = 0; e < NHALF; ++e) {
          // (sacc8 holds sum (p * scale - W))
          float bq = bacc[cs][e] + __shfl_xor(bacc[cs][e], 16);
          bq += __shfl_xor(bq, 32);
          float sq8 = sacc8[cs][e] + __shfl_xor(sacc8[cs][e], 16);
          sq8 += __shfl_xor(sq8, 32);
          bsum[e] = fmaf(8.0f, sq8, bq);
        }
      }
      float lsum = l_run[cs] + __shfl_xor(l_run[cs], 16);
      lsum += __shfl_xor(lsum, 32);
      const int hp = cs * kHeadSlots + hse;  // the column's head in the chunk
#pragma unroll
      for (int c = 0; c < NC; ++c) {
        // lane (col, qe) holds dims 4 (16 c + 4 qe + i) + k, of group
        // (64 (c % 2) + 16 qe) / G of their half; its column's slot stands for
        // that group when gse % NGH equals it, and of the NS / NGH copies of a
        // group copy r writes rows qe with qe (NS / NGH) / 4 == r
        constexpr int R = NS / NGH;
        if (gse % NGH == (64 * (c & 1) + 16 * qe) / G && gse / NGH == (qe * R) / 4) {
          const float bg = bsum[(c >> 1) < NHALF ? (c >> 1) : 0];
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            // (code sums times 2^20, the operands' code scale)
            const float4 o4 = make_float4(fmaf(acc_o[cs][c][0][i], 1048576.0f, bg),
                                          fmaf(acc_o[cs][c][1][i], 1048576.0f, bg),
                                          fmaf(acc_o[cs][c][2][i], 1048576.0f, bg),
                                          fmaf(acc_o[cs][c][3][i], 1048576.0f, bg));
            *reinterpret_cast<float4*>(part + hp * D + 4 * (16 * c + 4 * qe + i)) = o4;
          }
        }
      }
      if (lane_e < kHeadSlots) {
        part_m[cs * kHeadSlots + lane_e] = m_run[cs];
        part_l[cs * kHeadSlots + lane_e] = lsum;
      }
    }
  }
  __syncthreads();

  {
    const float* base = reinterpret_cast<const float*>(smem[0][0]);
    constexpr int kWaveFloats = kStages * kStageBytes / 4;
    const int lane_e = lane_id_volatile();
    for (int o = wave * 64 + lane_e; o < nh * D; o += kThreads) {
      const int h = o / D, dd = o % D;
      float mw[kWaves];
      float M = kMinit;
#pragma unroll
      for (int w = 0; w < kWaves; ++w) {
        mw[w] = base[w * kWaveFloats + kChunk * D + h];
        M = fmaxf(M, mw[w]);
      }
      float num = 0.0f, den = 0.0f;
#pragma unroll
      for (int w = 0; w < kWaves; ++w) {
        const float* pw = base + w * kWaveFloats;
        const float f = __builtin_amdgcn_exp2f(mw[w] - M);
        num = fmaf(f, pw[h * D + dd], num);
        den = fmaf(f, pw[kChunk * D + kChunk + h], den);
      }
      // agent-scope stores write through to the device-coherent level, so the
      // block that combines (on any XCD) reads them without a cache flush
      float* rec = ws + (((size_t)b * Hq + (h0 + h)) * max_splits + split) * (D + 4);
      __hip_atomic_store(&rec[dd], (den > 0.0f) ? num / den : 0.0f, __ATOMIC_RELAXED,
                         __HIP_MEMORY_SCOPE_AGENT);
      if (dd == 0) {
        __hip_atomic_store(&rec[D], M, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_store(&rec[D + 1], den, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
    }
  }

  // ---- the last split of this (request, KV head, head chunk) to finish
  // combines all of them (log-sum-exp), so no second kernel is needed.
  // Ordering: every word the blocks exchange is accessed with device-scope
  // atomic instructions on both sides.  The records are written by
  // agent-scope atomic stores (global_store sc1: written through to the
  // device-coherent level) and read by device-scope coherent loads
  // (buffer_load sc1, the instruction of an agent-scope atomic load: no
  // non-coherent cached copy is returned).  Each thread waits until its
  // record stores have completed (vmcnt 0) before the barrier that precedes
  // the ticket increment, a device-scope atomic; the combining block issues
  // its record loads only after it has seen the last ticket (in-order issue,
  // no speculation).  The compiler's release and acquire for this exchange
  // are the same instructions plus an L2 write-back before the increment
  // and an L2 invalidation after it, which only matter for data written or
  // read without device-scope atomics (there is none here); in every block
  // they cost ~2.5 us per call at 262,144 positions.
  wait_vm<0>();     // this thread's records are stored
  __syncthreads();  // ... and every thread's; the merge buffers are free
  uint32_t* ticket = tickets + ((size_t)b * Hkv + kv) * n_hchunks + hc;
  if (tid == 0)
    s_ticket = __hip_atomic_fetch_add(ticket, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  __syncthreads();
  if (s_ticket != (uint32_t)(S - 1)) return;
  if (tid == 0) __hip_atomic_store(ticket, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  combine_splits<D, (kChunk < kWaves ? kWaves / kChunk : 1), kWaves>(ws, out, b, Hq, sq, h0, nh,
                                                                        max_splits, S);
}

template <int D, int G, bool APPEND, int CS>
hipError_t launch_cs(const jf_kv_layout& L, const jf_kv_pool_ptrs& pool, const void* k_new,
                     const void* v_new, const void* q,
                     int32_t B, int32_t Hq, const int32_t* bt, int32_t max_pages,
                     const int32_t* lens, float scale, int32_t max_splits, uint32_t* tickets,
                     float* records, void* out, int32_t sq, hipStream_t stream) {
  const int gq = Hq / L.num_kv_heads;
  constexpr int kChunk = head_slots<D, G>() * CS;
  const int n_hchunks = (gq + kChunk - 1) / kChunk;
  // Splits per request: enough blocks for one per CU when one request runs
  // alone, at most max_splits.  The count does not depend on the batch (a
  // request's output is bitwise the same in any batch) nor on the lengths
  // (they are on the device).
  const int64_t per_split = (int64_t)L.num_kv_heads * n_hchunks;
  const int split_cap =
      (int)std::max<int64_t>(1, std::min<int64_t>(max_splits, jfkv::num_cus() / per_split));
  // several head chunks: one x index per (split, KV head, chunk), grouped by
  // XCD (the kernel decodes it)
  const int64_t slots = (int64_t)split_cap * L.num_kv_heads;
  dim3 grid = n_hchunks == 1
                  ? dim3(split_cap, L.num_kv_heads, B)
                  : dim3((uint32_t)(((slots + kXcds - 1) / kXcds) * kXcds * n_hchunks), 1, B);
  hipLaunchKernelGGL((decode_kernel<D, G, APPEND, CS>), grid, dim3(64 * waves_for<D>()), 0, stream,
                     static_cast<uint8_t*>(pool.k_codes), static_cast<uint32_t*>(pool.k_meta),
                     static_cast<uint8_t*>(pool.v_codes), static_cast<uint32_t*>(pool.v_meta),
                     static_cast<const uint4*>(k_new), static_cast<const uint4*>(v_new),
                     static_cast<const __half*>(q),
                     bt, lens, records, tickets, static_cast<__half*>(out), Hq, (int)sq,
                     L.num_kv_heads, L.page_size, L.num_pages, max_pages, max_splits, split_cap,
                     n_hchunks,
                     scale * kLog2e);
  return hipGetLastError();
}

// Two column sets per block where one would leave query heads of the KV head
// for a second chunk (more heads than head_slots, as in the short verifier,
// whose heads are query heads times tokens); head_dim 256 keeps one set (its
// accumulators fill the registers).
template <int D, int G, bool APPEND>
hipError_t launch_t(const jf_kv_layout& L, const jf_kv_pool_ptrs& pool, const void* k_new,
                    const void* v_new, const void* q,
                    int32_t B, int32_t Hq, const int32_t* bt, int32_t max_pages,
                    const int32_t* lens, float scale, int32_t max_splits, uint32_t* tickets,
                    float* records, void* out, int32_t sq, hipStream_t stream) {
  if constexpr (D <= 128) {
    if (Hq / L.num_kv_heads > head_slots<D, G>())
      return launch_cs<D, G, APPEND, 2>(L, pool, k_new, v_new, q, B, Hq, bt, max_pages, lens,
                                         scale, max_splits, tickets, records, out, sq, stream);
  }
  return launch_cs<D, G, APPEND, 1>(L, pool, k_new, v_new, q, B, Hq, bt, max_pages, lens, scale,
                                    max_splits, tickets, records, out, sq, stream);
}

}  // namespace

namespace jfkv {

// Compute units of the current device (queried once per device).
int num_cus() {
  constexpr int kMaxDevices = 64;
  static int cached[kMaxDevices] = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) return 256;
  if (dev < kMaxDevices && cached[dev] > 0) return cached[dev];
  int n = 0;
  if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
    n = 256;
  if (dev < kMaxDevices) cached[dev] = n;
  return n;
}

namespace {
hipError_t dispatch(const jf_kv_layout& L, const jf_kv_pool_ptrs& pool, const void* k_new,
                    const void* v_new, const void* q, int32_t B, int32_t Hq, const int32_t* bt,
                    int32_t max_pages, const int32_t* lens, float scale, int32_t max_splits,
                    uint32_t* tickets, float* records, void* out, int32_t sq,
                    hipStream_t stream) {
#define JF_ARGS L, pool, k_new, v_new, q, B, Hq, bt, max_pages, lens, scale, max_splits, tickets, \
                records, out, sq, stream
#define JF_CASE(D_, G_)                                              \
  if (L.head_dim == D_ && L.group_size == G_)                        \
    return k_new ? launch_t<D_, G_, true>(JF_ARGS) : launch_t<D_, G_, false>(JF_ARGS);
  JF_CASE(64, 32)
  JF_CASE(64, 64)
  JF_CASE(128, 32)
  JF_CASE(128, 64)
  JF_CASE(128, 128)
  JF_CASE(256, 32)
  JF_CASE(256, 64)
  JF_CASE(256, 128)
#undef JF_CASE
#undef JF_ARGS
  return hipErrorInvalidValue;
}
}  // namespace

hipError_t launch_decode(const jf_kv_layout& L, const jf_kv_pool_ptrs& pool, const void* k_new,
                         const void* v_new, const void* q, int32_t B, int32_t Hq,
                         const int32_t* bt, int32_t max_pages, const int32_t* lens, float scale,
                         int32_t max_splits, void* ws, void* out, hipStream_t stream,
                         int32_t sq) {
  // completion counters first, then the split records
  uint32_t* tickets = static_cast<uint32_t*>(ws);
  float* records = reinterpret_cast<float*>(static_cast<uint8_t*>(ws) + kDecodeCounterBytes);
  return dispatch(L, pool, k_new, v_new, q, B, Hq, bt, max_pages, lens, scale, max_splits,
                  tickets, records, out, sq, stream);
}

// ---- the decode step without a caller workspace: its completion counters
// and split records live in `scratch`, one copy per device, addressed through
// hipGetSymbolAddress once per device.  The counters must start at zero: a
// small fill kernel clears them on the first call on each device (every call
// that completes leaves them zero again).
namespace {
__global__ void zero_words(uint32_t* p, int n) {
  for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x)
    p[i] = 0u;
}
}  // namespace

hipError_t static_scratch(void** out, bool* first_use) {
  constexpr int kMaxDevices = 64;
  static std::mutex mu;
  static void* ptrs[kMaxDevices] = {};
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(mu);
  *first_use = ptrs[dev] == nullptr;
  if (*first_use) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    ptrs[dev] = p;
  }
  *out = ptrs[dev];
  return hipSuccess;
}

hipError_t launch_decode_static(const jf_kv_layout& L, const jf_kv_pool_ptrs& pool,
                                const void* k_new, const void* v_new, const void* q, int32_t B,
                                int32_t Hq, const int32_t* bt, int32_t max_pages,
                                const int32_t* lens, float scale, int32_t max_splits, void* out,
                                hipStream_t stream) {
  void* base = nullptr;
  bool first = false;
  hipError_t e = static_scratch(&base, &first);
  if (e != hipSuccess) return e;
  uint32_t* tickets = static_cast<uint32_t*>(base);
  float* records = reinterpret_cast<float*>(static_cast<uint8_t*>(base) + kStaticTicketBytes);
  if (first) {
    hipLaunchKernelGGL(zero_words, dim3(16), dim3(256), 0, stream, tickets,
                       (int)(kStaticTicketBytes / sizeof(uint32_t)));
    if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  return dispatch(L, pool, k_new, v_new, q, B, Hq, bt, max_pages, lens, scale, max_splits,
                  tickets, records, out, 1, stream);
}

}  // namespace jfkv
