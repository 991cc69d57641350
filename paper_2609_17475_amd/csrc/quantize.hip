// Quantize-and-append of new K/V rows into 4-bit pages (gfx950).
//
// Encoding: group-wise affine 4-bit codes with an fp16 scale and bias per
// group of head_dim elements (the affine 4-bit format the paper's
// Introduction describes for weights), written into 256-token pages
// through the request's page table (Background, "Compact histories need
// reusable storage").  The contract is bit-exact; every binary32 step is a
// separately rounded IEEE operation in the order given in include/jfkv.h.
//
// Group extremes are exact and independent of the element order (IEEE
// minimum/maximum of fp16 values and integer total-order keys of their bit
// patterns, -0 below +0); the mapping of rows to waves and lanes is described
// at each kernel.
#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>

#include <algorithm>

#include "jfkv_internal.h"
#include "jfkv_quant.h"

#pragma clang fp contract(off)

namespace {

using jfkv::quantize8;
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
// Row staging of the tiled kernel: a 1 KiB load block plus 16 bytes, so the
// lanes reading 128-byte row slices spread over the LDS banks.
constexpr int kStagePitch = 1040;
// a where mask is set, else b (bitwise; keeps register arrays out of memory).
__device__ __forceinline__ uint32_t pick(uint32_t mask, uint32_t a, uint32_t b) {
  return (a & mask) | (b & ~mask);
}
// fl32(x - b) for the fp16 value x in half H of word w, given nb = -b: one
// mixed-precision FMA, x * 1 + nb, so a single rounding as in a binary32
// subtraction.
template <int H>
__device__ __forceinline__ float sub_half(uint32_t w, float nb) {
  float r;
  if constexpr (H == 0)
    asm("v_fma_mix_f32 %0, %1, 1.0, %2 op_sel_hi:[1,0,0]" : "=v"(r) : "v"(w), "v"(nb));
  else
    asm("v_fma_mix_f32 %0, %1, 1.0, %2 op_sel:[1,0,0] op_sel_hi:[1,0,0]" : "=v"(r) : "v"(w), "v"(nb));
  return r;
}
// floor(x) as an integer (v_cvt_flr_i32_f32).
__device__ __forceinline__ int cvt_flr(float x) {
  int r;
  asm("v_cvt_flr_i32_f32 %0, %1" : "=v"(r) : "v"(x));
  return r;
}
__device__ __forceinline__ uint32_t order_key(uint32_t h) { return jfkv::q_order_key(h); }
__device__ __forceinline__ uint32_t from_key(uint32_t k) { return jfkv::q_from_key(k); }
__device__ __forceinline__ float h2f(uint32_t bits) { return jfkv::q_h2f(bits); }
__device__ __forceinline__ uint32_t f2h_up_pos(float x) { return jfkv::q_f2h_up_pos(x); }

// Latency-oriented kernel for small appends (a decode step's rows): one
// group of G elements is handled by G/8 consecutive lanes, each holding 8
// fp16 values (one 16-byte load); min and max reduce over the group's lanes
// with cross-lane swaps; each lane packs its 8 codes into one 32-bit word
// (one store for K, two 16-bit stores for the position-paired V layout).
__global__ __launch_bounds__(256) void quantize_small_kernel(
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
  // codes and (scale, bias) of the lane's 8 values; the group's lpg lanes
  // (aligned runs) exchange its minimum and maximum
  uint32_t meta_word;
  const uint32_t packed = quantize8(x, lpg, meta_word);
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

  const int64_t ph = (int64_t)page * Hkv + kv;  // (page, kv head) run
  jfkv::store_codes8(kind ? v_codes : k_codes, kind ? v_meta : k_meta, kind != 0, ph, P, D, G,
                     slot, c8, lpg, packed, meta_word);
}

// Appends of at least this many rows use the row-tiled kernel below.
constexpr int32_t kTiledMinRows = 256;

// Margin of the reciprocal shortcut for the code rint(r), r = fl(d / s):
// with inv = v_rcp_f32(s) (within 1 ulp) and t = fma(d, inv, 0.5) (one
// rounding), |d inv - d/s| <= |d/s| 2^-23 <= 2^-19 and the fma adds at most
// 2^-21 for t < 16, while |r - d/s| <= 2^-21; so |t - (r + 0.5)| < 2^-17.
// Whenever t is farther than 2^-15 from every integer, r + 0.5 lies strictly
// between the same two integers (r is no tie), and floor(t) = rint(r)
// exactly.  Codes whose t lies nearer an integer take the exact IEEE
// division instead.  (0 <= d/s <= 15 by construction of s, so t < 16.)
constexpr float kFracLo = 1.0f / 32768.0f;          // 2^-15 of margin
constexpr float kFracHi = 1.0f - 1.0f / 32768.0f;

// Row-tiled quantize-append.  A wave-tile is PW = 64 / (D/64) consecutive
// new rows of one KV head, K or V; lane (p, part) owns dims 64 part .. 64 part
// + 63 of row p of the tile, so when the rows are consecutive positions of
// one page (a bulk append) the wave's stores are contiguous runs: K codes
// 32 B per lane, V codes as whole 32-bit words of position pairs (the two
// rows of a pair swap halves by a lane exchange), (scale, bias) words per
// group.  Rows whose pair partner is not the neighbouring position (single
// rows, odd starts, page or request boundaries) store their V half-words
// alone.
//
// The grid is persistent: wave w takes tiles w, w + W, ... (W waves in the
// grid), and holds the next tile's rows in registers while it quantizes the
// current one, so every wave keeps a tile's loads in flight.  The loads
// cover whole rows (lane l fetches 16-byte chunk l % (D/8) of row l / (D/8)
// of each 1 KiB run); the wave passes them through its LDS stage to give
// each lane its 128-byte slice.
template <int D, int G>
__global__ __launch_bounds__(256) void quantize_rows_kernel(
    uint8_t* __restrict__ k_codes, uint32_t* __restrict__ k_meta,
    uint8_t* __restrict__ v_codes, uint32_t* __restrict__ v_meta,
    const uint4* __restrict__ k_new, const uint4* __restrict__ v_new,
    const int32_t* __restrict__ cu_tok, const int32_t* __restrict__ start_pos,
    const int32_t* __restrict__ block_tables, int32_t B, int32_t max_pages, int32_t total_tok,
    int32_t P, int32_t Hkv, int32_t NP, uint32_t n_tiles) {
  constexpr int LPR = D / 64;                 // lanes per row
  constexpr int PW = 64 / LPR;                // rows per wave-tile
  constexpr int NGL = (G >= 64) ? 1 : 64 / G;  // groups within a lane
  constexpr int EPG = (G >= 64) ? 64 : G;      // elements of a group within a lane
  constexpr int NG = D / G;
  constexpr int RPI = 512 / D;                // rows per 1 KiB load
  constexpr int CPR = D / 8;                  // 16-byte chunks per row
  const int lane = threadIdx.x & 63;
  const int wib = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // wave in block (scalar)
  const int64_t W = (int64_t)gridDim.x * (blockDim.x >> 6);
  const int p = lane / LPR, part = lane % LPR;
  __shared__ __attribute__((aligned(16))) uint8_t stage[4][8][kStagePitch];

  // Tile t = (row block * 2 + kind) * Hkv + kv: its rows as the loads cover
  // them (rows past the end re-read the last row; their results are not
  // stored).
  auto load_tile = [&](uint32_t kv, uint32_t rest, u32x4 (&v)[8]) {
    const int64_t r0 = (int64_t)(rest >> 1) * PW;
    const u32x4* src = reinterpret_cast<const u32x4*>((rest & 1) ? v_new : k_new) + kv * CPR + lane % CPR;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int64_t r = min(r0 + i * RPI + lane / CPR, (int64_t)total_tok - 1);
      v[i] = __builtin_nontemporal_load(src + r * Hkv * CPR);
    }
  };
  // Wave-uniform lookups of a tile's destination, in two steps so that each
  // step's loads return while the wave quantizes a tile: (1) the request lo
  // of its first row and that row's position; the tile is fast when it lies
  // in that request at positions >= 0, and then spans at most two pages (P
  // >= 64 >= PW); (2) the IDs of those pages.
  struct Dest {
    int32_t lo, pos0, lp_a, lp_b, pg_a, pg_b;
    bool fast;
  };
  auto dest_request = [&](uint32_t rest) {
    Dest d;
    const int64_t r0 = (int64_t)(rest >> 1) * PW;
    const int64_t r_last = min(r0 + PW, (int64_t)total_tok) - 1;
    int32_t lo = 0, hi = B;
    while (hi - lo > 1) {
      const int32_t mid = (lo + hi) >> 1;
      if (cu_tok[mid] <= r0) lo = mid; else hi = mid;
    }
    d.lo = lo;
    d.pos0 = start_pos[lo] + (int32_t)(r0 - cu_tok[lo]);
    d.fast = cu_tok[lo + 1] > r_last && d.pos0 >= 0;
    d.lp_a = d.pos0 / P;
    d.lp_b = (d.pos0 + (int32_t)(r_last - r0)) / P;  // lp_a or lp_a + 1
    d.pg_a = d.pg_b = -1;
    return d;
  };
  auto dest_pages = [&](Dest& d) {
    const int32_t* tb = block_tables + (int64_t)d.lo * max_pages;
    d.pg_a = (d.fast && d.lp_a < max_pages) ? tb[d.lp_a] : -1;
    d.pg_b = (d.fast && d.lp_b != d.lp_a && d.lp_b < max_pages) ? tb[d.lp_b] : -1;
  };

  const uint32_t Wn = gridDim.x * (blockDim.x >> 6);  // waves in the grid
  const uint32_t wq = Wn / Hkv, wr = Wn % Hkv;        // the step W in (rest, kv)
  uint32_t t = blockIdx.x * (blockDim.x >> 6) + wib;
  if (t >= n_tiles) return;  // wave-uniform
  uint32_t kv = t % Hkv, rest = t / Hkv;
  u32x4 nx[8];
  load_tile(kv, rest, nx);
  Dest nd = dest_request(rest);
  dest_pages(nd);
  for (;;) {
    // this tile's rows into the stage; the next tile's loads take their place
#pragma unroll
    for (int i = 0; i < 8; ++i)
      *reinterpret_cast<u32x4*>(&stage[wib][i][16 * lane]) = nx[i];
    const Dest cd = nd;
    const uint32_t ckv = kv, crest = rest;  // this tile's (kv and rest move on to the next)
    const bool more = (uint64_t)t + Wn < (uint64_t)n_tiles;
    if (more) {
      t += Wn;
      kv += wr;
      rest += wq;
      if (kv >= (uint32_t)Hkv) {
        kv -= Hkv;
        rest += 1;
      }
      load_tile(kv, rest, nx);
      nd = dest_request(rest);  // its pages: after this tile's codes
    }

    const int kind = (int)(crest & 1);
    const int64_t r0 = (int64_t)(crest >> 1) * PW;  // first row of the tile
    const int64_t row = r0 + p;
    const bool in_range = row < total_tok;

    // destination of the lane's row: page and slot (the fast case picks one
    // of the tile's two page IDs; otherwise the lane looks its row up)
    int32_t page = -1, slot = 0;
    if (cd.fast) {
      const int32_t pos = cd.pos0 + p;
      const bool second = pos >= (cd.lp_a + 1) * P;
      const int32_t pg = second ? cd.pg_b : cd.pg_a;
      if (in_range && pg >= 0 && pg < NP) {
        page = pg;
        slot = pos - (second ? cd.lp_a + 1 : cd.lp_a) * P;
      }
    } else if (in_range) {
      int32_t l2 = cd.lo, h2 = B;
      while (h2 - l2 > 1) {
        const int32_t mid = (l2 + h2) >> 1;
        if (cu_tok[mid] <= row) l2 = mid; else h2 = mid;
      }
      const int64_t pos = (int64_t)start_pos[l2] + (row - cu_tok[l2]);
      const int64_t lp = (pos >= 0) ? pos / P : -1;
      if (lp >= 0 && lp < max_pages) {
        const int32_t pg = block_tables[(int64_t)l2 * max_pages + lp];
        if (pg >= 0 && pg < NP) {
          page = pg;
          slot = (int32_t)(pos % P);
        }
      }
    }
    const bool valid = page >= 0;

    uint4 x[8];
    {
      const uint4* my = reinterpret_cast<const uint4*>(
          &stage[wib][p / RPI][(p % RPI) * 2 * D + 128 * part]);
#pragma unroll
      for (int i = 0; i < 8; ++i) x[i] = my[i];
    }

    uint32_t hw[32];  // the lane's 64 fp16 values, two per word
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      hw[4 * i] = x[i].x;
      hw[4 * i + 1] = x[i].y;
      hw[4 * i + 2] = x[i].z;
      hw[4 * i + 3] = x[i].w;
    }

    // group minimum and maximum: IEEE minimum/maximum of packed fp16 pairs
    // (exact, -0 below +0, so the same total order as the keys below; the
    // compiler folds them into three-input instructions), taken to integer
    // total-order keys (key = h ^ (sign ? 0xffff : 0x8000))
    uint32_t kmin[NGL], kmax[NGL];
#pragma unroll
    for (int gl = 0; gl < NGL; ++gl) {
      f16x2 lo2 = __builtin_bit_cast(f16x2, hw[gl * EPG / 2]), hi2 = lo2;
#pragma unroll
      for (int w = gl * EPG / 2 + 1; w < (gl + 1) * EPG / 2; ++w) {
        lo2 = __builtin_elementwise_minimum(lo2, __builtin_bit_cast(f16x2, hw[w]));
        hi2 = __builtin_elementwise_maximum(hi2, __builtin_bit_cast(f16x2, hw[w]));
      }
      lo2 = __builtin_elementwise_minimum(lo2, lo2.yx);
      hi2 = __builtin_elementwise_maximum(hi2, hi2.yx);
      kmin[gl] = order_key(__builtin_bit_cast(unsigned short, lo2.x));
      kmax[gl] = order_key(__builtin_bit_cast(unsigned short, hi2.x));
    }
    if constexpr (G == 128) {  // the group spans this lane and lane ^ 1
      kmin[0] = min(kmin[0], (uint32_t)__shfl_xor((int)kmin[0], 1));
      kmax[0] = max(kmax[0], (uint32_t)__shfl_xor((int)kmax[0], 1));
    }

    // scale and bias per group (the contract's steps, binary32 IEEE ops)
    uint32_t meta_w[NGL];
    float sf[NGL], bf[NGL], inv[NGL];
#pragma unroll
    for (int gl = 0; gl < NGL; ++gl) {
      const uint32_t mn_bits = from_key(kmin[gl]), mx_bits = from_key(kmax[gl]);
      const float mn = h2f(mn_bits), mx = h2f(mx_bits);
      const float range = __fsub_rn(mx, mn);
      const float step = __fdiv_rn(range, 15.0f);
      const uint32_t scale_bits = (range == 0.0f) ? 0u : f2h_up_pos(step);
      meta_w[gl] = scale_bits | (mn_bits << 16);  // bias = mn (exact in fp16)
      sf[gl] = h2f(scale_bits);
      bf[gl] = h2f(mn_bits);
      inv[gl] = (scale_bits == 0) ? 0.0f : __builtin_amdgcn_rcpf(sf[gl]);
    }

    // codes: floor(fma(d, 1/s, 0.5)) with d = fl(x - b), which is rint(fl(d /
    // s)) whenever t is not within 2^-15 of an integer (the margin above);
    // the extreme fractional parts are tracked so those codes can be redone
    float nb[NGL];
#pragma unroll
    for (int gl = 0; gl < NGL; ++gl) nb[gl] = -bf[gl];
    uint32_t cw[8];  // nibble i of word m = code of element 8m + i
    float fmin = 1.0f, fmax = 0.0f;
#pragma unroll
    for (int m = 0; m < 8; ++m) {
      uint32_t word = 0;
#pragma unroll
      for (int i = 0; i < 8; i += 2) {
        const int e = 8 * m + i, gl = e / EPG;
        const uint32_t w = hw[e >> 1];
        const float t0 = __builtin_fmaf(sub_half<0>(w, nb[gl]), inv[gl], 0.5f);
        const float t1 = __builtin_fmaf(sub_half<1>(w, nb[gl]), inv[gl], 0.5f);
        const float f0 = __builtin_amdgcn_fractf(t0), f1 = __builtin_amdgcn_fractf(t1);
        fmin = fminf(fmin, fminf(f0, f1));
        fmax = fmaxf(fmax, fmaxf(f0, f1));
        word |= (uint32_t)cvt_flr(t0) << (4 * i);
        word |= (uint32_t)cvt_flr(t1) << (4 * i + 4);
      }
      cw[m] = word;
    }
    if (__builtin_amdgcn_ballot_w64(fmin <= kFracLo || fmax >= kFracHi) != 0) {
      // some t lies near an integer: the exact IEEE division for those
      // elements (rare: each element index is redone only if a lane of the
      // wave needs it).  The values are passed through an empty asm so that
      // the quotients are recomputed here, not kept live from above.
      uint32_t hx[32];
#pragma unroll
      for (int w = 0; w < 32; ++w) {
        hx[w] = hw[w];
        asm volatile("" : "+v"(hx[w]));
      }
#pragma unroll
      for (int m = 0; m < 8; ++m) {
        uint32_t word = cw[m];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          const int e = 8 * m + i, gl = e / EPG;
          const float d = (i & 1) ? sub_half<1>(hx[e >> 1], nb[gl]) : sub_half<0>(hx[e >> 1], nb[gl]);
          const float f = __builtin_amdgcn_fractf(__builtin_fmaf(d, inv[gl], 0.5f));
          if (f <= kFracLo || f >= kFracHi) {
            uint32_t code = 0;
            if (sf[gl] != 0.0f) {
              const float r = __fdiv_rn(d, sf[gl]);
              code = (uint32_t)fminf(fmaxf(__builtin_rintf(r), 0.0f), 15.0f);
            }
            word = (word & ~(0xfu << (4 * i))) | (code << (4 * i));
          }
        }
        cw[m] = word;
      }
    }

    // V position pairs: both rows of a pair present and neighbours in one page?
    const int32_t partner_page = __shfl_xor(page, LPR);
    const int32_t partner_slot = __shfl_xor(slot, LPR);
    const bool odd = slot & 1;
    const uint32_t odd_mask = 0u - (uint32_t)odd;  // selects by mask: no indexed access to cw
    const bool paired = valid && partner_page == page && partner_slot == (slot ^ 1);
    uint32_t send[4], recv[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      send[i] = pick(odd_mask, cw[i], cw[4 + i]);  // the half-words the partner stores
      recv[i] = (uint32_t)__shfl_xor((int)send[i], LPR);
    }
    if (valid) {

    const int64_t ph = (int64_t)page * Hkv + ckv;  // (page, KV head) block
    if (kind == 0) {
      uint4* dst = reinterpret_cast<uint4*>(k_codes + (ph * P + slot) * (D / 2) + 32 * part);
      dst[0] = make_uint4(cw[0], cw[1], cw[2], cw[3]);
      dst[1] = make_uint4(cw[4], cw[5], cw[6], cw[7]);
    } else {
      // 4-dim chunk u = 16 part + i of the lane: half-word i of cw (16 bits)
      uint8_t* vbase = v_codes + ph * P * (D / 2) + (int64_t)(slot >> 1) * (D / 4) * 4;
      if (paired) {
        // even row: words u = 16 part + 0..7, odd row: 16 part + 8..15; word
        // u = (even row's chunk) | (odd row's chunk) << 16
        uint32_t wv[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) {
          const uint32_t mine = pick(odd_mask, cw[4 + i / 2], cw[i / 2]) >> (16 * (i & 1)) & 0xffffu;
          const uint32_t other = recv[i / 2] >> (16 * (i & 1)) & 0xffffu;
          wv[i] = odd ? (other | (mine << 16)) : (mine | (other << 16));
        }
        uint4* dst = reinterpret_cast<uint4*>(vbase + (16 * part + (odd ? 8 : 0)) * 4);
        dst[0] = make_uint4(wv[0], wv[1], wv[2], wv[3]);
        dst[1] = make_uint4(wv[4], wv[5], wv[6], wv[7]);
      } else {
        uint16_t* dst = reinterpret_cast<uint16_t*>(vbase + (16 * part) * 4 + (slot & 1) * 2);
#pragma unroll
        for (int i = 0; i < 16; ++i) dst[2 * i] = (uint16_t)(cw[i / 2] >> (16 * (i & 1)));
      }
    }
    uint32_t* meta = (kind ? v_meta : k_meta) + (ph * P + slot) * NG;
    if constexpr (G == 32) {
      *reinterpret_cast<uint2*>(meta + 2 * part) = make_uint2(meta_w[0], meta_w[1]);
    } else if constexpr (G == 64) {
      meta[part] = meta_w[0];
    } else {
      if ((part & 1) == 0) meta[part / 2] = meta_w[0];
    }
    }  // valid
    if (!more) break;
    dest_pages(nd);
  }
}

}  // namespace

namespace jfkv {

hipError_t launch_quantize_append(const jf_kv_layout& L, const jf_kv_pool_ptrs& pool,
                                  const void* k_new, const void* v_new,
                                  const int32_t* cu_tok, const int32_t* start_pos,
                                  const int32_t* block_tables, int32_t B, int32_t max_pages,
                                  int32_t total_tok, hipStream_t stream) {
  if (total_tok < kTiledMinRows) {  // a few rows: 8 elements per lane, shortest latency
    const int64_t lanes = (int64_t)total_tok * 2 * L.num_kv_heads * (L.head_dim / 8);
    const int64_t blocks = (lanes + 255) / 256;
    hipLaunchKernelGGL(quantize_small_kernel, dim3((uint32_t)blocks), dim3(256), 0, stream,
                       static_cast<uint8_t*>(pool.k_codes), static_cast<uint32_t*>(pool.k_meta),
                       static_cast<uint8_t*>(pool.v_codes), static_cast<uint32_t*>(pool.v_meta),
                       static_cast<const uint4*>(k_new), static_cast<const uint4*>(v_new), cu_tok,
                       start_pos, block_tables, B, max_pages, total_tok, L.page_size,
                       L.num_kv_heads, L.head_dim, L.group_size, L.num_pages);
    return hipGetLastError();
  }
  const int pw = 64 / (L.head_dim / 64);  // rows per wave-tile
  const int64_t tiles = ((int64_t)total_tok + pw - 1) / pw * 2 * L.num_kv_heads;
  // persistent: four blocks of four waves per CU (the LDS stages allow four)
  if (tiles > 0xffffffffLL) return hipErrorInvalidValue;  // (beyond any device's memory)
  const int64_t blocks = std::min<int64_t>((tiles + 3) / 4, (int64_t)jfkv::num_cus() * 4);
#define JF_Q_ARGS                                                                          \
  static_cast<uint8_t*>(pool.k_codes), static_cast<uint32_t*>(pool.k_meta),                \
      static_cast<uint8_t*>(pool.v_codes), static_cast<uint32_t*>(pool.v_meta),            \
      static_cast<const uint4*>(k_new), static_cast<const uint4*>(v_new), cu_tok, start_pos, \
      block_tables, B, max_pages, total_tok, L.page_size, L.num_kv_heads, L.num_pages,       \
      (uint32_t)tiles
#define JF_Q_CASE(D_, G_)                                                                 \
  if (L.head_dim == D_ && L.group_size == G_) {                                           \
    hipLaunchKernelGGL((quantize_rows_kernel<D_, G_>), dim3((uint32_t)blocks), dim3(256), 0, \
                       stream, JF_Q_ARGS);                                                \
    return hipGetLastError();                                                             \
  }
  JF_Q_CASE(64, 32)
  JF_Q_CASE(64, 64)
  JF_Q_CASE(128, 32)
  JF_Q_CASE(128, 64)
  JF_Q_CASE(128, 128)
  JF_Q_CASE(256, 32)
  JF_Q_CASE(256, 64)
  JF_Q_CASE(256, 128)
#undef JF_Q_CASE
#undef JF_Q_ARGS
  return hipErrorInvalidValue;
}

}  // namespace jfkv
