/*
 * diffkv_oracle.h -- plain, slow, serial CPU reference for the DiffKV hot path.
 *
 * TEST INFRASTRUCTURE ONLY.  Only tests/, the smoke check and the CPU-baseline
 * leg of the benchmark may load this library.  It shares no code, header,
 * table or constant generator with the GPU library under
 * paper_2412_03131_amd/csrc/; both implement the page layout independently
 * from its written description.
 *
 * What it follows (DiffKV, arXiv 2412.03131):
 *   - asymmetric min/max quantization with fp16 scale/zero (Sec. 2.2),
 *     applied per 32-dim group, keys at more bits than values (Sec. 4);
 *   - three-level token classing, quota form and the sequence-length
 *     adaptive threshold form (Sec. 4, prompt phase, and Algorithm 1);
 *   - the generation-phase policy of Algorithm 1 (candidate leaving the
 *     recent window, victims, re-quantization to the low precision);
 *   - unified pages, circular free page list, bidirectional page table and
 *     the prefix-sum allocation/recycling schedule (Sec. 5.2, 5.3);
 *   - softmax attention, Eq. (1) of Sec. 2.1, evaluated in fp64 over the
 *     dequantized cache, and the split-sequence merge (Sec. 6.2);
 *   - the significance scores (Sec. 4): the running mean of the attention
 *     probability each kept token receives, maximum over a KV head's query
 *     heads, updated once per decode step.
 *
 * Every function is serial and state changes happen in the order the text
 * describes; there is no blocking, fusion or reordering.
 *
 * Parity pins: see tests/test_oracle_*.py.  All functions are pinned.
 */
#ifndef DIFFKV_ORACLE_H
#define DIFFKV_ORACLE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum { DKO_HIGH = 0, DKO_LOW = 1 };
enum { DKO_CLASS_PRUNE = -1 };

/* sticky device-status bits, same meaning as the GPU library's */
enum { DKO_ST_OUT_OF_PAGES = 1u, DKO_ST_TABLE_OVERFLOW = 2u };

/* ---- fp16 <-> fp32 by bit manipulation (IEEE binary16, RNE) ---------- */
float    dko_half_to_float(uint16_t h);
uint16_t dko_float_to_half(float f);
void     dko_half_to_float_n(int64_t n, const uint16_t* h, float* f);
void     dko_float_to_half_n(int64_t n, const float* f, uint16_t* h);

/* ---- one quantization group (Sec. 2.2) --------------------------------
 * x: n fp16 bit patterns; bits: code width.  Outputs the fp16 scale and
 * zero-point bit patterns and one code per element (one byte each).       */
void dko_quantize_group(const uint16_t* x, int n, int bits,
                        uint16_t* scale, uint16_t* zero, uint8_t* codes);

/* ---- layout ------------------------------------------------------------ */
typedef struct dko_layout {
    int32_t head_dim, group;
    int32_t k_bits[2], v_bits[2];
    int32_t tokens_per_page[2];
    int32_t max_seq_len, p_max;
    int64_t page_bytes;
    int32_t off_kcode[2], off_kmeta[2], off_vcode[2], off_vmeta[2];
    int32_t off_score[2], off_pos[2], used_bytes[2];
} dko_layout;

/* returns 0 on success, nonzero if the parameters do not describe a layout */
int dko_layout_init(dko_layout* L, int head_dim, int group,
                    const int32_t k_bits[2], const int32_t v_bits[2],
                    const int32_t tokens_per_page[2], int max_seq_len);

/* ---- cache state (all host arrays) ------------------------------------ */
typedef struct dko_cache {
    uint8_t*  pool;       /* [num_pages][page_bytes]                        */
    int64_t   num_pages;
    int32_t*  table;      /* [num_tables][p_max], -1 = empty slot            */
    int32_t*  pages;      /* [num_tables][2] pages held per section          */
    int32_t*  len;        /* [num_tables][2] tokens held per section         */
    int32_t*  seq_len;    /* [num_seqs] logical tokens seen (incl. pruned)   */
    int32_t*  ring;       /* [num_pages] circular free page list             */
    int64_t*  ring_ptr;   /* [2] {head (allocation), tail (recycling)}       */
    uint32_t* status;     /* [1] sticky bits                                 */
    int32_t   num_seqs, num_kv_heads;
} dko_cache;

/* ---- classing (Sec. 4) ------------------------------------------------
 * One table's new tokens.  score[j] for j < n.  Quota form if quota != NULL
 * ({n_hi, n_lo}), threshold form otherwise with N = seq_len after the
 * append.  The last `window` tokens are high precision and outside the
 * quotas.  cls[j] = DKO_HIGH, DKO_LOW or DKO_CLASS_PRUNE.                 */
void dko_classify(int n, const float* score, const int32_t* quota,
                  float alpha_h, float alpha_l, int seq_len_after,
                  int window, int8_t* cls);

/* ---- allocation (Sec. 5.2) ------------------------------------------- */
int dko_alloc_pages(const dko_layout* L, dko_cache* C, int num_tables,
                    const int32_t* demand /* [num_tables][2] */);

/* ---- quantize + place (Sec. 4 compressor, Sec. 5.2 unified pages) ----
 * new_len[b] tokens per sequence, packed: token j of sequence b is row
 * new_off(b)+j of k/v ([rows][Hkv][D] fp16) and score ([rows][Hkv]).
 * Returns 0; failures are reported in *status with the state unchanged.   */
int dko_quantize_append(const dko_layout* L, dko_cache* C,
                        const int32_t* new_len,
                        const uint16_t* k, const uint16_t* v,
                        const float* score, const int32_t* quota,
                        float alpha_h, float alpha_l, int window);

/* ---- free-list compaction (Sec. 5.2, 5.3) ---------------------------- */
int dko_compact(const dko_layout* L, dko_cache* C, int num_tables,
                const uint8_t* release /* [num_tables][p_max] */);

/* ---- generation phase (Sec. 4, Algorithm 1) ---------------------------
 * One decode step's policy for every table, after the step's append put the
 * newest token into the high section (the recent window of W positions).
 * Candidate: the high token at position seq_len - 1 - W.  Thresholds
 * alpha_h/N, alpha_l/N (fp32, N = seq_len).  Victims: lowest score (ties:
 * lowest position) outside the window.  Removal moves a section's last
 * token into the hole and clears the vacated slot; a token entering the low
 * section is re-quantized (fp32 fmaf dequantization, fp16 RNE, low-precision
 * quantization) and appended, or takes the slot of the low victim it
 * evicts.  A low section that grows past its pages takes one page from the
 * ring (all-or-nothing across tables).  Returns 0; failures set *status.  */
int dko_generation_step(const dko_layout* L, dko_cache* C, float alpha_h, float alpha_l,
                        int window);

/* ---- page decoding ----------------------------------------------------
 * Dequantized key/value of section token u of table t (fp64, exact).     */
void dko_read_token(const dko_layout* L, const dko_cache* C, int t, int sec,
                    int u, double* k_hat, double* v_hat,
                    float* score, int32_t* pos);

/* ---- attention, Eq. (1), fp64 ----------------------------------------
 * q: [B][Hq][D] fp16.  out: [B][Hq][D], lse: [B][Hq] (may be NULL).
 * Query head hq reads KV head hq / (Hq/Hkv).  Tokens: the high-precision
 * section, then the low-precision section.  Empty head: out 0, lse -inf. */
int dko_attention(const dko_layout* L, const dko_cache* C, int num_q_heads,
                  const uint16_t* q, double sm_scale,
                  double* out, double* lse);

/* Partial state of one page range [p0, p1) of the unified list (high
 * pages first, then low pages) for one (b, hq): m = max logit, l = sum of
 * exp(logit - m), acc[D] = sum of exp(logit - m) * v_hat.                 */
void dko_attention_partial(const dko_layout* L, const dko_cache* C,
                           int num_q_heads, const uint16_t* q,
                           double sm_scale, int b, int hq, int p0, int p1,
                           double* m, double* l, double* acc);
/* Merge S partials (Sec. 6.2 sequence split): out and lse of one head.   */
void dko_merge_partials(int S, int D, const double* m, const double* l,
                        const double* acc, double* out, double* lse);

/* ---- memory accounting against an FP16 cache (Sec. 1, Fig. 1) -------
 * Fraction of FP16 key bits and value bits used by a head holding n_hi
 * high-precision and n_lo low-precision tokens out of n_total.           */
/* Significance update of one decode step (Sec. 4): after the step's query
 * q (one per sequence and query head) has attended the compressed cache, every
 * kept token of table t = b*H + h receives one more attention score.  Its
 * score is the mean of the scores received so far, a score being the largest
 * softmax probability of the token among the g query heads of KV head h
 * (softmax over the table's kept tokens, logits sm_scale * q . k_hat, fp64).
 * A token at position p of a sequence of N = seq_len[b] tokens has then
 * received N - p scores (queries p .. N-1), so its stored fp32 score s
 * becomes s + (x - s) / (N - p), evaluated in fp64 and rounded to fp32.
 * Returns 1 when num_q_heads is not a multiple of H. */
int dko_update_significance(const dko_layout* L, dko_cache* C, int num_q_heads,
                            const uint16_t* q, double sm_scale);
/* Prompt-phase significance of every prompt token (Sec. 4): q [rows][Hq][D],
 * k [rows][Hkv][D] fp16 bits, rows concatenated per sequence (new_len[B]);
 * score [rows][Hkv] fp32 out; select [B][Hkv] or NULL.  1 on bad shapes. */
int dko_prompt_significance(int B, const int32_t* new_len, int num_q_heads, int num_kv_heads,
                            int D, const uint16_t* q, const uint16_t* k, double sm_scale,
                            const uint8_t* select, float* score);
/* Scores (fp64) of the last m tokens of one N-token prompt for KV head h; q
 * and k point at the prompt's first row.  1 on bad arguments. */
int dko_prompt_significance_tail(int N, int num_q_heads, int num_kv_heads, int D, const uint16_t* q,
                                 const uint16_t* k, double sm_scale, int h, int m, double* score_tail);

void dko_kv_bits_fraction(const dko_layout* L, int n_hi, int n_lo,
                          int n_total, double* k_frac, double* v_frac);

#ifdef __cplusplus
}
#endif
#endif
