// Single-query decode attention over TQ4 pages (d = 256), split-K with the
// same bounded workspace and in-kernel combine as the affine decode.
//
// TQ4 (Sec. 3.1, eq. codec; Appendix A, Table codec) stores a vector x as an
// fp16 norm rho^ and 256 4-bit indices z into 16 shared centroids c, with
// x^ = rho^ S H c[z] / 16 (H the unnormalised Hadamard matrix of order 256,
// S the diagonal of random signs).  By linearity the rotation leaves the page
// scan:
//   q . x^_t = rho^_t (q' . c[z_t])          with q' = H S q / 16 (once),
//   o = sum_t p_t x^_t / sum_t p_t = S H u / (16 sum_t p_t),
//        u = sum_t p_t rho^_t c[z_t]           (rotated back once).
// So the scan reads the packed indices and the norms where they are stored
// (page-native, Sec. 3.1) and never reconstructs a vector.
//
// Each byte of packed indices becomes the fp16 centroids of its two indices
// by one LDS read from a 256-entry table of centroid pairs (entry e: c[e % 16]
// in the low half, c[e / 16] in the high half), shared by every query head of
// the KV head: for keys the pair is directly an operand word (dims 2j, 2j + 1
// of one position); for values two reads and a permute give one dim at two
// positions.  The table is held 64 times, interleaved so that lane l reads
// copy l from its own bank (random entries would otherwise collide in the LDS
// banks), and 64 KiB-aligned, so that one byte permute of the index word
// forms a lookup's address (the index byte is the address's second byte).
// The table's 64 KiB hold q' before the page loop and the final rotation
// after it.  The centroids are rounded to fp16 once (relative error
// <= 2^-11); q' enters as an fp16 high part plus an fp16 low part.
//
// Matrix-core layout (v_mfma_f32_16x16x32_f16; lane (m, q4) = (lane % 16,
// lane / 16) feeds operand row m, k-slots 8 q4 .. 8 q4 + 7, and receives
// column m, rows 4 q4 .. 4 q4 + 3 of the result):
//   scores  S^T[pos][head] over 8 k-steps of 32 dims, two 16-position tiles
//           per 32-position row; tile t row m is position 8 (m / 4) + 4 t +
//           m % 4, and k-step kb of lane quarter q4 is index word 8 q4 + kb
//           (dims 0..7 of the word in order), so each lane's K data is 32
//           contiguous bytes of one position and its scores are positions
//           8 q4 .. 8 q4 + 7;
//   values  u^T[dim][head] += c[z][dim][pos] x W[pos][head], W = p rho^_V
//           (fp16); product j (0..15) has row m = dim 16 m + j, so lane
//           (m, q4) holds index words 2 m, 2 m + 1 of positions 8 q4 ..
//           8 q4 + 7 (8 bytes each) and the k-slots are exactly the positions
//           of its own scores; byte b of those words holds dims 16 m + 2 b
//           and + 1 of one position.
// Two waves per SIMD (eight per block): the table reads' latency of one wave
// is covered by the other's work.
// Online softmax per head with a lazy running maximum (raised only when a
// logit exceeds it by more than 2 in log2 units, so p <= 4).
#include <hip/hip_fp16.h>
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <algorithm>

#include "jfkv.h"
#include "jfkv_internal.h"

namespace {

typedef _Float16 h8 __attribute__((ext_vector_type(8)));
typedef _Float16 h2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

// Device-coherent (sc1) buffer loads of one head's split records (256
// values, then m and l); the resource covers that head's max_splits records,
// so the hardware also bounds-checks every access.
constexpr int kCpolSc1 = 16;
__device__ __forceinline__ __amdgpu_buffer_rsrc_t head_records(const float* base, int max_splits) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<float*>(base), (short)0,
                                           max_splits * (256 + 4) * 4, 0x00020000);
}

// Streaming loads of page data (non-temporal: read once per call).
__device__ __forceinline__ uint4 ld_nt(const uint32_t* p) {
  const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
  return make_uint4(v.x, v.y, v.z, v.w);
}
__device__ __forceinline__ uint2 ld_nt2(const uint32_t* p) {
  const u32x2 v = __builtin_nontemporal_load(reinterpret_cast<const u32x2*>(p));
  return make_uint2(v.x, v.y);
}

constexpr int kD = 256;           // head dimension of the format
constexpr int kWordsPerVec = kD / 8;
constexpr int kWaves = 8;         // two waves per SIMD, one block per CU
constexpr int kParts = 4;         // per-wave partial buffers (waves w and w + 4 merge first)
constexpr int kThreads = 64 * kWaves;
constexpr int kRowPos = 32;       // positions per row (two 16-position tiles)
constexpr int kMaxCols = 16;      // query heads per KV head: one column block
constexpr float kLog2e = 1.4426950408889634f;
constexpr float kTau = 2.0f;      // lazy-rescale margin, log2 units
constexpr float kMinit = -1e30f;  // finite initial maximum (masked rows give p = 0)
constexpr int kMaxSplits = 256;   // split cap of the launch (the combine's LDS bound)

__device__ __forceinline__ f32x4 mfma(h8 a, h8 b, f32x4 c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
}

// In-place Walsh-Hadamard transform (unnormalised, natural order) of n rows
// of 256 floats in LDS, by the whole block.
__device__ void fwht_rows(float* x, int n) {
  for (int h = 1; h < kD; h <<= 1) {
    for (int i = threadIdx.x; i < n * (kD / 2); i += kThreads) {
      const int r = i / (kD / 2), k = i % (kD / 2);
      float* row = x + r * kD;
      const int a = (k / h) * (2 * h) + (k % h);
      const float u = row[a], v = row[a + h];
      row[a] = u + v;
      row[a + h] = u - v;
    }
    __syncthreads();
  }
}

// Page-aligned split s of n_pages pages into S parts (remainder first).
__device__ __forceinline__ void split_range(int n_pages, int S, int s, int& pb, int& pe) {
  const int base = n_pages / S, rem = n_pages % S;
  pb = s * base + min(s, rem);
  pe = pb + base + (s < rem ? 1 : 0);
}

// One row's data in registers.
struct RowBuf {
  uint4 k[2][2];    // tile t: index words 8 q4 .. 8 q4 + 7 of the tile's position
  uint2 v[8];       // words 2 m, 2 m + 1 of positions 8 q4 + p
  uint4 kn, vn;     // norms of positions 8 q4 .. 8 q4 + 7
  bool ok;          // the row's page exists
};

__global__ __launch_bounds__(kThreads) void tq4_decode_kernel(
    const uint32_t* __restrict__ k_words, const __half* __restrict__ k_norms,
    const uint32_t* __restrict__ v_words, const __half* __restrict__ v_norms,
    const float* __restrict__ k_signs, const float* __restrict__ v_signs,
    const float* __restrict__ centroids, const __half* __restrict__ q,
    const int32_t* __restrict__ block_tables, const int32_t* __restrict__ seq_lens,
    float* __restrict__ ws, uint32_t* __restrict__ tickets, __half* __restrict__ out, int Hq,
    int Hkv, int P, int NP, int max_pages, int max_splits, int split_cap, float scale_log2) {
  // index byte -> fp16 centroids of its nibbles, 64 copies (the page loop);
  // before and after the loop the same bytes hold q' and the final rotation
  __shared__ __attribute__((aligned(65536))) uint32_t s_tab[256 * 64];
  float* const s_x = reinterpret_cast<float*>(s_tab);     // [kMaxCols][kD]
  static_assert(kMaxCols * kD <= 256 * 64, "q' fits the table's bytes");
  __shared__ float s_part[kParts][kMaxCols * (kD + 2)];  // per-wave partials (u, m, l)
  __shared__ h8 s_qop[8][2][64];                         // score B operands (q' high, low)
  __shared__ uint32_t s_ticket;

  const int split = blockIdx.x, kv = blockIdx.y, b = blockIdx.z;
  const int gq = Hq / Hkv;
  const int h0 = kv * gq;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int l16 = lane & 15, q4 = lane >> 4;

  const int L = min(seq_lens[b], max_pages * P);
  if (L <= 0) {  // an empty request: zero output rows, written by split 0
    if (split == 0)
      for (int i = tid; i < gq * kD; i += kThreads)
        out[((size_t)b * Hq + h0) * kD + i] = __float2half(0.0f);
    return;
  }
  const int n_pages = (L + P - 1) / P;
  const int S = min(split_cap, n_pages);
  if (split >= S) return;
  int pb, pe;
  split_range(n_pages, S, split, pb, pe);
  const int t_end = min(pe * P, L);

  // ---- q' = H S q / 16 per query head (a negative scale negates it)
  const float qsign = scale_log2 < 0.0f ? -1.0f : 1.0f;
  for (int i = tid; i < gq * kD; i += kThreads) {
    const int h = i / kD, d = i % kD;
    s_x[i] = qsign * k_signs[d] * __half2float(q[((size_t)b * Hq + h0 + h) * kD + d]);
  }
  __syncthreads();
  fwht_rows(s_x, gq);
  // B operands in LDS (one 16-byte entry per lane, read back conflict-free):
  // k-step kb, lane (col, q4): word 8 q4 + kb, dims 0..7 of it, as an
  // fp16 high part and an fp16 low part; each wave fills one k-step
#pragma unroll
  for (int k2 = 0; k2 < 8 / kWaves; ++k2) {
    const int kb = (8 / kWaves) * wave + k2;
    const int w = 8 * q4 + kb;
    const bool col_on = l16 < gq;
    h8 hi, lo;
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int d = 8 * w + e;
      const float v = s_x[min(l16, gq - 1) * kD + d] * 0.0625f;
      const _Float16 vh = col_on ? (_Float16)v : (_Float16)0.0f;
      hi[e] = vh;
      lo[e] = col_on ? (_Float16)(v - (float)vh) : (_Float16)0.0f;
    }
    s_qop[kb][0][lane] = hi;
    s_qop[kb][1][lane] = lo;
  }
  __syncthreads();  // q' is in the operands: its bytes become the table
  // pair table: entry e holds c[e & 15] (low half) and c[e >> 4] (high half),
  // copy c (0..63) at word 64 e + c
  for (int i = tid; i < 256 * 64; i += kThreads) {
    const int e = i >> 6;
    const uint32_t lo = __builtin_bit_cast(uint16_t, (_Float16)centroids[e & 15]);
    const uint32_t hi = __builtin_bit_cast(uint16_t, (_Float16)centroids[e >> 4]);
    s_tab[i] = lo | (hi << 16);
  }
  __syncthreads();
  const float kfold = fmaxf(fabsf(scale_log2), 1e-30f);  // |scale| in log2 units

  // ---- this wave's rows: split rows wave, wave + kWaves, ...
  const int rpp = P / kRowPos;  // rows per page
  const int n_split_pages = pe - pb;
  const int split_rows = n_split_pages * rpp;
  const int my_rows = split_rows > wave ? (split_rows - wave + kWaves - 1) / kWaves : 0;
  const size_t head_slots = (size_t)P;  // vectors per (page, KV head)
  // page IDs of the split, 64 per register (lane k: page pb + 64 g + k)
  int grp = -1, pg_reg = -1;
  auto page_of = [&](int pi) {
    const int g = pi >> 6;
    if (g != grp) {
      grp = g;
      const int k = 64 * g + lane;
      pg_reg = (k < n_split_pages) ? block_tables[(size_t)b * max_pages + pb + k] : -1;
    }
    return __builtin_amdgcn_readlane(pg_reg, pi & 63);
  };

  auto load_row = [&](int r, RowBuf& rb) {
    const int R = wave + kWaves * r;
    const int pi = R / rpp, rs = R % rpp;
    int page = page_of(pi);
    rb.ok = (unsigned)page < (unsigned)NP;
    if (!rb.ok) page = 0;  // never read outside the pool; the row is masked
    const size_t vec0 = ((size_t)page * Hkv + kv) * head_slots + (size_t)rs * kRowPos;
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      const int pos = 8 * (l16 >> 2) + 4 * t + (l16 & 3);
      const uint32_t* src = k_words + (vec0 + pos) * kWordsPerVec + 8 * q4;
      rb.k[t][0] = ld_nt(src);
      rb.k[t][1] = ld_nt(src + 4);
    }
#pragma unroll
    for (int p = 0; p < 8; ++p) rb.v[p] = ld_nt2(v_words + (vec0 + 8 * q4 + p) * kWordsPerVec + 2 * l16);
    rb.kn = ld_nt(reinterpret_cast<const uint32_t*>(k_norms + vec0 + 8 * q4));
    rb.vn = ld_nt(reinterpret_cast<const uint32_t*>(v_norms + vec0 + 8 * q4));
  };

  // Lane l reads copy l (its own bank): the LDS address of entry e is
  // base + 256 e + 4 l with the table 64 KiB-aligned, i.e. the base's bytes
  // 2..3, the index byte itself as byte 1 and 4 l as byte 0, which one byte
  // permute assembles.
  const uint32_t lane4 = (uint32_t)(uintptr_t)s_tab + 4u * (uint32_t)lane;
  // (k, the byte of the word, is a constant once the loops are unrolled)
  auto lookup = [&](uint32_t word, uint32_t k) {
    const uint32_t a = __builtin_amdgcn_perm(word, lane4, 0x03020000u | ((4u + k) << 8));
    return *reinterpret_cast<const __attribute__((address_space(3))) uint32_t*>(a);
  };
  f32x4 acc_v[16];
#pragma unroll
  for (int j = 0; j < 16; ++j) acc_v[j] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
  float m_run = kMinit, thr = kMinit, l_run = 0.0f;
  const h2 ones = {(_Float16)1.0f, (_Float16)1.0f};

  auto compute_row = [&](const RowBuf& rb, int r) {
    const int R = wave + kWaves * r;
    const int t_row = (pb + R / rpp) * P + (R % rpp) * kRowPos;  // first logical position
    // ---- scores
    float sc[8];  // positions 8 q4 + 4 t + i at index 4 t + i
    const uint32_t kn[4] = {rb.kn.x, rb.kn.y, rb.kn.z, rb.kn.w};
    const uint32_t w[2][8] = {{rb.k[0][0].x, rb.k[0][0].y, rb.k[0][0].z, rb.k[0][0].w,
                               rb.k[0][1].x, rb.k[0][1].y, rb.k[0][1].z, rb.k[0][1].w},
                              {rb.k[1][0].x, rb.k[1][0].y, rb.k[1][0].z, rb.k[1][0].w,
                               rb.k[1][1].x, rb.k[1][1].y, rb.k[1][1].z, rb.k[1][1].w}};
    f32x4 acc[2] = {{0.0f, 0.0f, 0.0f, 0.0f}, {0.0f, 0.0f, 0.0f, 0.0f}};
#pragma unroll
    for (int kb = 0; kb < 8; ++kb) {
      const h8 qh = s_qop[kb][0][lane], ql = s_qop[kb][1][lane];
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        const uint32_t x = w[t][kb];
        const u32x4 r = {lookup(x, 0), lookup(x, 1), lookup(x, 2), lookup(x, 3)};
        const h8 a = __builtin_bit_cast(h8, r);
        acc[t] = mfma(a, qh, acc[t]);
        acc[t] = mfma(a, ql, acc[t]);
      }
    }
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int k = 4 * t + i;
        const _Float16 rho = __builtin_bit_cast(h2, kn[k >> 1])[k & 1];
        sc[k] = acc[t][i] * (float)rho;
      }
    uint32_t vn[4] = {rb.vn.x, rb.vn.y, rb.vn.z, rb.vn.w};
    const bool full = rb.ok && t_row + kRowPos <= t_end;  // wave-uniform
    if (!full) {
      asm volatile("" ::: "memory");  // keep the masking behind the branch
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const bool ok = rb.ok && t_row + 8 * q4 + k < t_end;
        sc[k] = ok ? sc[k] : -INFINITY;
        if (!ok) {  // a masked position contributes nothing (its norm may be anything)
          h2 pr = __builtin_bit_cast(h2, vn[k >> 1]);
          pr[k & 1] = (_Float16)0.0f;
          vn[k >> 1] = __builtin_bit_cast(uint32_t, pr);
        }
      }
    }
    // ---- online softmax (one running maximum per head: lanes of one column)
    float mx = sc[0];
#pragma unroll
    for (int k = 1; k < 8; ++k) mx = fmaxf(mx, sc[k]);
    mx *= kfold;
    if (__builtin_amdgcn_ballot_w64(mx > thr) != 0) {
      float M = fmaxf(mx, __shfl_xor(mx, 16));
      M = fmaxf(M, __shfl_xor(M, 32));
      if (M > m_run) {
        const float alpha = __builtin_amdgcn_exp2f(m_run - M);
        m_run = M;
        thr = M + kTau;
        l_run *= alpha;
#pragma unroll
        for (int j = 0; j < 16; ++j) acc_v[j] *= alpha;
      }
    }
    u32x4 Wv;  // W = p rho^_V, positions 8 q4 + 0 .. 7 in k-slot order
#pragma unroll
    for (int k2 = 0; k2 < 4; ++k2) {
      const h2 p = {(_Float16)__builtin_amdgcn_exp2f(fmaf(sc[2 * k2], kfold, -m_run)),
                    (_Float16)__builtin_amdgcn_exp2f(fmaf(sc[2 * k2 + 1], kfold, -m_run))};
      l_run = __builtin_amdgcn_fdot2(p, ones, l_run, false);
      Wv[k2] = __builtin_bit_cast(uint32_t, p * __builtin_bit_cast(h2, vn[k2]));
    }
    const h8 W = __builtin_bit_cast(h8, Wv);
    // ---- values: product j has row m = dim 16 m + j
#pragma unroll
    for (int bb = 0; bb < 8; ++bb) {
      // centroid pairs (low, high nibble of byte bb) of the eight positions
      uint32_t t[8];
#pragma unroll
      for (int p = 0; p < 8; ++p) {
        const uint32_t word = (bb < 4) ? rb.v[p].x : rb.v[p].y;
        t[p] = lookup(word, bb & 3);
      }
#pragma unroll
      for (int hn = 0; hn < 2; ++hn) {  // low nibble: dim 16 m + 2 bb; high: + 1
        const uint32_t sel = hn ? 0x07060302u : 0x05040100u;
        const u32x4 a = {__builtin_amdgcn_perm(t[1], t[0], sel), __builtin_amdgcn_perm(t[3], t[2], sel),
                         __builtin_amdgcn_perm(t[5], t[4], sel), __builtin_amdgcn_perm(t[7], t[6], sel)};
        const int j = 2 * bb + hn;
        acc_v[j] = mfma(__builtin_bit_cast(h8, a), W, acc_v[j]);
      }
    }
  };

  RowBuf b0, b1;
  if (my_rows > 0) load_row(0, b0);
  for (int r = 0; r < my_rows; r += 2) {
    if (r + 1 < my_rows) load_row(r + 1, b1);
    compute_row(b0, r);
    if (r + 1 < my_rows) {
      if (r + 2 < my_rows) load_row(r + 2, b0);
      compute_row(b1, r + 1);
    }
  }

  // ---- merge the waves: each writes its unnormalised u^T (lane (col, q4):
  // dims 64 q4 + 16 i + j), its maximum and its row sum
  {
    float lsum = l_run + __shfl_xor(l_run, 16);
    lsum += __shfl_xor(lsum, 32);
    // waves 4..7 write their partials; waves 0..3 fold their own into them
    float* part = s_part[wave & (kParts - 1)];
    if (wave >= kParts && l16 < gq) {
#pragma unroll
      for (int j = 0; j < 16; ++j)
#pragma unroll
        for (int i = 0; i < 4; ++i) part[l16 * (kD + 2) + 64 * q4 + 16 * i + j] = acc_v[j][i];
      if (q4 == 0) {
        part[l16 * (kD + 2) + kD] = m_run;
        part[l16 * (kD + 2) + kD + 1] = lsum;
      }
    }
    __syncthreads();
    if (wave < kParts && l16 < gq) {
      const float mo = part[l16 * (kD + 2) + kD], lo = part[l16 * (kD + 2) + kD + 1];
      const float M = fmaxf(m_run, mo);
      const float f = __builtin_amdgcn_exp2f(m_run - M), fo = __builtin_amdgcn_exp2f(mo - M);
#pragma unroll
      for (int j = 0; j < 16; ++j)
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          float* u = &part[l16 * (kD + 2) + 64 * q4 + 16 * i + j];
          *u = fmaf(f, acc_v[j][i], fo * *u);
        }
      if (q4 == 0) {
        part[l16 * (kD + 2) + kD] = M;
        part[l16 * (kD + 2) + kD + 1] = fmaf(f, lsum, fo * lo);
      }
    }
  }
  __syncthreads();
  for (int o = tid; o < gq * kD; o += kThreads) {
    const int h = o / kD, d = o % kD;
    float mw[kParts], M = kMinit;
#pragma unroll
    for (int w = 0; w < kParts; ++w) {
      mw[w] = s_part[w][h * (kD + 2) + kD];
      M = fmaxf(M, mw[w]);
    }
    float num = 0.0f, den = 0.0f;
#pragma unroll
    for (int w = 0; w < kParts; ++w) {
      const float f = __builtin_amdgcn_exp2f(mw[w] - M);
      num = fmaf(f, s_part[w][h * (kD + 2) + d], num);
      den = fmaf(f, s_part[w][h * (kD + 2) + kD + 1], den);
    }
    float* rec = ws + (((size_t)b * Hq + h0 + h) * max_splits + split) * (kD + 4);
    __hip_atomic_store(&rec[d], den > 0.0f ? num / den : 0.0f, __ATOMIC_RELAXED,
                       __HIP_MEMORY_SCOPE_AGENT);
    if (d == 0) {
      __hip_atomic_store(&rec[kD], M, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      __hip_atomic_store(&rec[kD + 1], den, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }

  // ---- the last split of (request, KV head) to finish combines them all
  // (log-sum-exp over the splits, in the rotated space), then rotates back.
  // Ordering: every word the blocks exchange is accessed with device-scope
  // atomic instructions on both sides: the records are written by
  // agent-scope atomic stores (global_store sc1, written through to the
  // device-coherent level) and read by device-coherent loads (buffer_load
  // sc1).  Each thread waits until its record stores have completed before
  // the barrier that precedes the ticket increment, a device-scope atomic;
  // the combining block issues its record loads only after it has seen the
  // last ticket.  A release/acquire pair would add an L2 write-back before
  // the increment and an invalidation after it, which matter only for data
  // exchanged without device-scope atomics (there is none).
  __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0): this thread's records are stored
  __syncthreads();
  uint32_t* ticket = tickets + (size_t)b * Hkv + kv;
  if (tid == 0)
    s_ticket = __hip_atomic_fetch_add(ticket, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  __syncthreads();
  if (s_ticket != (uint32_t)(S - 1)) return;
  if (tid == 0) __hip_atomic_store(ticket, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  // split weights w_s = l_s 2^(m_s - M) (M the largest m_s of a non-empty
  // split) and their sum, one wave per head, lanes over the splits; kept in
  // LDS (s_part reused: gq * S <= 16 * kMaxSplits = 4,096 weights, then the
  // gq sums)
  float* s_w = s_part[0];                   // [gq][S]
  float* s_den = s_part[0] + kMaxCols * kMaxSplits;  // [gq]
  static_assert(kMaxCols * kMaxSplits + kMaxCols <= kMaxCols * (kD + 2), "weights fit");
  for (int h = wave; h < gq; h += kWaves) {
    const auto rs = head_records(ws + ((size_t)b * Hq + h0 + h) * max_splits * (kD + 4), max_splits);
    float mv[kMaxSplits / 64], lv[kMaxSplits / 64];
    float M = -INFINITY;
#pragma unroll
    for (int j = 0; j < kMaxSplits / 64; ++j) {
      const int s = lane + 64 * j;
      const f32x2 ml = s < S ? __builtin_amdgcn_raw_buffer_load_b64(rs, (s * (kD + 4) + kD) * 4, 0, kCpolSc1)
                             : f32x2{0.0f, 0.0f};
      mv[j] = ml.y > 0.0f ? ml.x : -INFINITY;
      lv[j] = ml.y;
      M = fmaxf(M, mv[j]);
    }
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) M = fmaxf(M, __shfl_xor(M, off));
    float den = 0.0f;
#pragma unroll
    for (int j = 0; j < kMaxSplits / 64; ++j) {
      const int s = lane + 64 * j;
      const float w = mv[j] == -INFINITY ? 0.0f : lv[j] * __builtin_amdgcn_exp2f(mv[j] - M);
      if (s < S) s_w[h * S + s] = w;
      den += w;
    }
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) den += __shfl_xor(den, off);
    if (lane == 0) s_den[h] = den;
  }
  __syncthreads();
  // o = sum_s w_s o_s / sum_s w_s.  A wave task is (head, half of the dims);
  // lane (c, k) = (lane % 32, lane / 32) sums dims 128 half + 4 c .. + 3 over
  // the splits k, k + 2, ..., kCh independent 16-byte record loads at a time
  constexpr int kCh = 32;
  for (int task = wave; task < 2 * gq; task += kWaves) {
    const int h = task >> 1, k = lane >> 5;
    const int d0 = (kD / 2) * (task & 1) + 4 * (lane & 31);
    const auto rs = head_records(ws + ((size_t)b * Hq + h0 + h) * max_splits * (kD + 4), max_splits);
    float4 acc = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
    for (int s0 = k; s0 < S; s0 += 2 * kCh) {
      f32x4 o[kCh];
#pragma unroll
      for (int i = 0; i < kCh; ++i) {  // past the end: a valid record, weight 0
        const int s = min(s0 + 2 * i, S - 1);
        o[i] = __builtin_amdgcn_raw_buffer_load_b128(rs, (s * (kD + 4) + d0) * 4, 0, kCpolSc1);
      }
#pragma unroll
      for (int i = 0; i < kCh; ++i) {
        const int s = s0 + 2 * i;
        const float w = s < S ? s_w[h * S + s] : 0.0f;
        acc.x = fmaf(w, o[i].x, acc.x);
        acc.y = fmaf(w, o[i].y, acc.y);
        acc.z = fmaf(w, o[i].z, acc.z);
        acc.w = fmaf(w, o[i].w, acc.w);
      }
    }
    acc.x += __shfl_xor(acc.x, 32);
    acc.y += __shfl_xor(acc.y, 32);
    acc.z += __shfl_xor(acc.z, 32);
    acc.w += __shfl_xor(acc.w, 32);
    if (k == 0) {
      const float den = s_den[h];
      const float inv = den > 0.0f ? 1.0f / den : 0.0f;
      s_x[h * kD + d0 + 0] = acc.x * inv;
      s_x[h * kD + d0 + 1] = acc.y * inv;
      s_x[h * kD + d0 + 2] = acc.z * inv;
      s_x[h * kD + d0 + 3] = acc.w * inv;
    }
  }
  __syncthreads();
  fwht_rows(s_x, gq);
  for (int o = tid; o < gq * kD; o += kThreads) {
    const int h = o / kD, d = o % kD;
    out[((size_t)b * Hq + h0 + h) * kD + d] = __float2half(v_signs[d] * s_x[o] * 0.0625f);
  }
}

}  // namespace

namespace jfkv {

hipError_t launch_tq4_decode(const jf_kv_layout& L, const void* k_words, const void* k_norms,
                             const void* v_words, const void* v_norms, const float* k_signs,
                             const float* v_signs, const float* centroids, const void* q,
                             int32_t B, int32_t Hq, const int32_t* block_tables,
                             int32_t max_pages, const int32_t* seq_lens, float softmax_scale,
                             int32_t max_splits, void* ws, void* out, hipStream_t stream) {
  const int64_t per_split = L.num_kv_heads;
  const int split_cap = (int)std::max<int64_t>(
      1, std::min<int64_t>(std::min<int64_t>(max_splits, kMaxSplits),
                           (num_cus() + per_split - 1) / per_split));
  dim3 grid(split_cap, L.num_kv_heads, B);
  uint32_t* tickets = static_cast<uint32_t*>(ws);
  float* records = reinterpret_cast<float*>(static_cast<uint8_t*>(ws) + kDecodeCounterBytes);
  hipLaunchKernelGGL(tq4_decode_kernel, grid, dim3(kThreads), 0, stream,
                     static_cast<const uint32_t*>(k_words), static_cast<const __half*>(k_norms),
                     static_cast<const uint32_t*>(v_words), static_cast<const __half*>(v_norms),
                     k_signs, v_signs, centroids, static_cast<const __half*>(q), block_tables,
                     seq_lens, records, tickets, static_cast<__half*>(out), Hq,
                     L.num_kv_heads, L.page_size, L.num_pages, max_pages, max_splits, split_cap,
                     softmax_scale * kLog2e);
  return hipGetLastError();
}

}  // namespace jfkv
