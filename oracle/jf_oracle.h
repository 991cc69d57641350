/*
 * jf_oracle.h -- CPU oracle for attention over a group-wise 4-bit paged KV cache.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing on the product path may include, link,
 * load or call this code: only the test suite, the smoke check and the CPU
 * baseline leg of the benchmark do.  It shares no source with the HIP
 * library (no headers, helpers or constants); both sides implement the same
 * written definitions independently.
 *
 * What it computes (the paper being "JustFit: Just-in-Time State Management
 * for Local LLM Serving", KVExec component):
 *   - a paged KV pool of fixed-size token pages addressed through a
 *     per-request page table (Background, "Compact histories need reusable
 *     storage"; eq. kvbytes gives the per-position payload);
 *   - group-wise affine 4-bit codes with one fp16 scale and one fp16 bias per
 *     group (the affine 4-bit format the Introduction describes for
 *     weights: stored values plus scales and offsets), packed eight codes
 *     per 32-bit word (Appendix A, Table codec, per-vector storage);
 *   - exact softmax attention over the dequantized pages for single-query
 *     decode and for chunked prefill (Sec. 3.1 KVExec, "Decode and prefill
 *     need different kernels"; heads are independent, eq. groupattention).
 *
 * Floating point: the quantizer is an encoding and is fixed operation by
 * operation in IEEE binary32 (built with -ffp-contract=off, no fast-math);
 * attention is computed in binary64.  All fp16 values cross this interface
 * as uint16_t bit patterns.
 */
#ifndef JF_ORACLE_H
#define JF_ORACLE_H
#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct {
  int32_t page_size;    /* P: token positions per page                         */
  int32_t num_kv_heads; /* Hkv                                                  */
  int32_t head_dim;     /* d                                                    */
  int32_t group_size;   /* G: consecutive head_dim elements sharing scale/bias  */
  int32_t num_pages;    /* NP: pages in the pool                                */
} jfo_layout;

/* ---- fp16 bit-pattern helpers (binary16, IEEE 754-2008) ---------------- */
double   jfo_half_to_double(uint16_t h);
/* mode: 0 = round to nearest even, 1 = toward -inf, 2 = toward +inf */
uint16_t jfo_float_to_half(float f, int mode);
/* The same rounding of a binary64 value. */
uint16_t jfo_double_to_half(double x, int mode);

/* ---- one group ----------------------------------------------------------
 * x: G fp16 values.  Writes G unpacked codes (0..15), scale and bias bits. */
void jfo_quantize_group(const uint16_t* x, int32_t G, uint8_t* codes,
                        uint16_t* scale, uint16_t* bias);

/* n consecutive groups: x [n][G] -> codes [n][G], scales [n], biases [n]
 * (jfo_quantize_group on each; for tests that compare many groups). */
void jfo_quantize_groups(const uint16_t* x, int64_t n, int32_t G,
                         uint8_t* codes, uint16_t* scales, uint16_t* biases);

/* ---- pool byte layout ----------------------------------------------------
 * Per layer, one pool each for K and V:
 *   k_codes: uint8 [NP][Hkv][P][d/2]  row-major per position;
 *            byte j = code(2j) | code(2j+1) << 4.
 *   v_codes: uint8 [NP][Hkv][P/2][d/4][2][2]  positions paired (2s, 2s+1);
 *            for dims 4u..4u+3 of slot t, the two bytes at
 *            ((t/2)*(d/4) + u)*4 + (t%2)*2 hold
 *            code(4u) | code(4u+1)<<4, code(4u+2) | code(4u+3)<<4.
 *   *_meta:  fp16 [NP][Hkv][P][d/G][2] = (scale, bias) per group.
 * Byte offsets below are within one pool array. */
size_t jfo_codes_bytes(const jfo_layout* L);
size_t jfo_meta_elems(const jfo_layout* L);

/* Quantize and append n_tok rows per request.  k_new/v_new: fp16
 * [total_tok][Hkv][d]; request b owns rows cu_tok[b]..cu_tok[b+1]-1, written
 * at logical positions start_pos[b] + i through block_tables[b][.]
 * ([B][max_pages]).  Returns 0, or -1 on an out-of-range page reference. */
int jfo_quantize_append(const jfo_layout* L, uint8_t* k_codes, uint16_t* k_meta,
                        uint8_t* v_codes, uint16_t* v_meta,
                        const uint16_t* k_new, const uint16_t* v_new,
                        const int32_t* cu_tok, const int32_t* start_pos,
                        const int32_t* block_tables, int32_t B,
                        int32_t max_pages);

/* Dequantize the vector stored at (page, kv head, slot): out[d] in fp64. */
void jfo_dequant_vector(const jfo_layout* L, const uint8_t* codes,
                        const uint16_t* meta, int is_v, int32_t page,
                        int32_t kv, int32_t slot, double* out);

/* Page -> operand reconstruction of KV heads kv0 .. kv0+g-1 over logical
 * positions 0..n-1 of one request (table: [max_pages]): binary16 bits
 * out[g][n][d], each element the exact dequantized value rounded to nearest
 * (ties to even); pages outside [0, num_pages) give zeros.  Returns 0, or
 * -1 for invalid arguments. */
int jfo_reconstruct(const jfo_layout* L, const uint8_t* codes, const uint16_t* meta, int is_v,
                    const int32_t* table, int32_t max_pages, int32_t n, int32_t kv0, int32_t g,
                    uint16_t* out);

/* Single-query decode for B requests.  q: fp16 [B][Hq][d].  Request b
 * attends to its logical positions 0..seq_lens[b]-1.  out: fp64 [B][Hq][d].
 * Returns 0, or -1 on invalid arguments. */
int jfo_decode(const jfo_layout* L, const uint8_t* k_codes,
               const uint16_t* k_meta, const uint8_t* v_codes,
               const uint16_t* v_meta, const uint16_t* q, int32_t B,
               int32_t Hq, const int32_t* block_tables, int32_t max_pages,
               const int32_t* seq_lens, double alpha, double* out);

/* Chunked prefill for one request.  q: fp16 [T][Hq][d]; k_chunk/v_chunk:
 * fp16 [T][Hkv][d].  Query i sits at absolute position prefix_len + i and
 * attends to the dequantized prefix 0..prefix_len-1 (through block_table)
 * and to chunk rows 0..i.  chunk_quantized = 0 uses the chunk's fp16 rows as
 * they are; 1 uses their quantize->dequantize round trip.  rows (n_rows
 * entries, or NULL for all T) selects which query rows to compute; out is
 * fp64 [n_rows][Hq][d] in the order of rows. */
int jfo_prefill(const jfo_layout* L, const uint8_t* k_codes,
                const uint16_t* k_meta, const uint8_t* v_codes,
                const uint16_t* v_meta, const uint16_t* q,
                const uint16_t* k_chunk, const uint16_t* v_chunk, int32_t T,
                int32_t Hq, const int32_t* block_table, int32_t max_pages,
                int32_t prefix_len, double alpha, int chunk_quantized,
                const int32_t* rows, int32_t n_rows, double* out);

/* Threads the OpenMP loops use (1 when built without OpenMP), and a way to
 * set it (for timing the oracle on one core and on all of them). */
int jfo_max_threads(void);
void jfo_set_threads(int n);

#ifdef __cplusplus
}
#endif
#endif
