/*
 * diffkv.h -- C ABI of the DiffKV decode hot path for AMD Instinct MI355X
 * (gfx950).  DiffKV: arXiv 2412.03131, "Differentiated Memory Management
 * for Large Language Models with Parallel KV Compaction".
 *
 * What the library computes
 *   A differentiated, paged KV cache: keys are kept at more bits than values
 *   (K8V4 for high-precision tokens, K4V2 for low-precision tokens, Sec. 4),
 *   each token is kept high, kept low or pruned by its significance score
 *   (Sec. 4), and every (sequence, KV head) pair -- a "table" -- keeps its own
 *   number of tokens of each kind.  Memory is managed with unified pages, a
 *   circular free page list and bidirectional page tables (Sec. 5.2); decode
 *   attention reads the compressed pages directly (Sec. 6.2).
 *
 * Conventions
 *   - All entry points are C, take plain pointers and sizes, never allocate,
 *     free or synchronise, and keep no state between calls (except the
 *     per-device scratch address of diffkv_decode_attention_noalloc).
 *   - "device" pointers point to GPU memory of the current HIP device;
 *     "host" pointers to CPU memory.  The caller owns every buffer.
 *   - `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *     All work is enqueued on it and the call returns immediately.  Calls
 *     on one cache must be ordered on one stream; different caches are
 *     independent.
 *   - Return value: host-detectable errors (bad arguments, unsupported
 *     layout, small workspace, launch failure).  On any non-OK return
 *     nothing was enqueued (except DIFFKV_E_LAUNCH, which reports that an
 *     enqueue failed).
 *   - Device-detected conditions set sticky bits in *cache->status (device
 *     word, never cleared by the library).  The operations that can set them
 *     are all-or-nothing: when a bit is raised by a call, that call changed
 *     nothing in the cache.  The caller reads the word after a sync and
 *     recovers (e.g. releases finished sequences through compaction, then
 *     retries), and clears it.
 *   - fp16 values are passed as IEEE binary16 bit patterns (uint16_t).
 */
#ifndef DIFFKV_H
#define DIFFKV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t diffkv_status;
enum {
    DIFFKV_OK = 0,
    DIFFKV_E_INVAL = 1,       /* null pointer, negative or inconsistent size       */
    DIFFKV_E_UNSUPPORTED = 2, /* layout/shape the gfx950 kernels do not implement  */
    DIFFKV_E_WORKSPACE = 3,   /* ws_bytes smaller than diffkv_workspace_size()     */
    DIFFKV_E_LAUNCH = 4,      /* a HIP launch or runtime call failed               */
    DIFFKV_E_SCRATCH = 5      /* the call needs more than the fixed scratch of
                                 diffkv_decode_attention_noalloc                   */
};

/* sticky bits of *diffkv_cache.status */
enum {
    DIFFKV_ST_OUT_OF_PAGES = 1u,   /* the free region (tail - head) was too small     */
    DIFFKV_ST_TABLE_OVERFLOW = 2u, /* a table would hold more than p_max pages        */
    DIFFKV_ST_BAD_INPUT = 4u       /* new_len disagreed with total_new / max_new      */
};

enum { DIFFKV_HIGH = 0, DIFFKV_LOW = 1 };

/*
 * Page layout (Sec. 5.2, "unified pages").  Every page has the same byte
 * stride; its precision is fixed when a table takes it.  A page of
 * precision p holds T = tokens_per_page[p] tokens in six segments, in this
 * order, each starting on a 64-byte boundary of the page:
 *   K codes   [head_dim*k_bits/128 chunks][T][16 B]: chunk c holds dims
 *             c*(128/k_bits) .. +128/k_bits-1 of one token, element e at
 *             bit e*k_bits of the 16 bytes;
 *   K meta    [T][head_dim/group] {fp16 scale, fp16 zero};
 *   V codes   [head_dim][T*v_bits/8 B]: token slot s of dim d at bit s*v_bits
 *             of the dim's row;
 *   V meta    [head_dim/group][T] {fp16 scale, fp16 zero};
 *   scores    [T] fp32 (significance score as given);
 *   positions [T] int32 (token position in its sequence).
 * Bits are little-endian within bytes.  page_bytes = the larger of the two
 * precisions' sizes.  A fresh page (one whose slot 0 is being written) is
 * cleared first, so unused slots are zero bytes.
 * Table width p_max = ceil(max_seq_len / tokens_per_page[HIGH]) + 1: one
 * more than the paper's max_len / T_high, since a partial high page and a
 * partial low page can coexist.
 */
typedef struct diffkv_layout {
    int32_t head_dim, group;
    int32_t k_bits[2], v_bits[2];      /* [HIGH], [LOW]                       */
    int32_t tokens_per_page[2];        /* [HIGH], [LOW]                       */
    int32_t max_seq_len, p_max;
    int64_t page_bytes;
    int32_t off_kcode[2], off_kmeta[2], off_vcode[2], off_vmeta[2];
    int32_t off_score[2], off_pos[2], used_bytes[2];
} diffkv_layout;

/*
 * Cache state (all device memory, all caller-owned).  Table t = b*num_kv_heads
 * + h is the bidirectional page table of sequence b, KV head h (Sec. 5.2):
 * high-precision page IDs grow from slot 0 to the right, low-precision page
 * IDs from slot p_max-1 to the left; empty slots hold -1.  Token u of a
 * section lives in slot u % T of the section's page u / T; appends add
 * tokens in position order (a generation step's removal then moves a
 * section's last token into the hole).  The free page list is a ring of
 * num_pages IDs; the free IDs are ring[head % n .. tail % n) with head/tail
 * monotone int64 counters (start pointer allocates, end pointer recycles).
 */
typedef struct diffkv_cache {
    uint8_t*  pool;          /* device [num_pages][page_bytes]                     */
    int64_t   num_pages;
    int32_t*  page_table;    /* device [num_tables][p_max]                         */
    int32_t*  pages;         /* device [num_tables][2] pages held per section      */
    int32_t*  len;           /* device [num_tables][2] tokens held per section     */
    int32_t*  seq_len;       /* device [num_seqs] tokens seen per sequence (incl.
                                pruned); the threshold form's N                   */
    int32_t*  ring;          /* device [num_pages] circular free page list         */
    int64_t*  ring_ptr;      /* device [2] {head, tail}; tail - head = free pages  */
    uint32_t* status;        /* device [1] sticky DIFFKV_ST_* bits                 */
    int32_t   num_seqs;      /* B                                                  */
    int32_t   num_kv_heads;  /* Hkv; num_tables = B * Hkv                          */
} diffkv_cache;

/* Fill *out (host) from the parameters: segment offsets, page_bytes, p_max.
 * Bits must be 1, 2, 4 or 8, head_dim*k_bits a multiple of 128,
 * T*v_bits a multiple of 8, tokens_per_page[LOW] >= tokens_per_page[HIGH].
 * DIFFKV_E_INVAL otherwise.  Any valid layout is accepted here.  The append,
 * attention and significance kernels implement head_dim 128, group 32 and
 * these (high | low) section formats (precision levels of Sec. 4 and
 * Sec. 7.2), DIFFKV_E_UNSUPPORTED otherwise:
 *   K8V4, 16 tokens | K4V2, 32 tokens   (the paper's two levels)
 *   K8V8, 16 tokens | K4V2, 32 tokens
 *   K8V2, 16 tokens | K4V1, 32 tokens
 *   K8V4, 16 tokens | K4V2, 16 tokens
 * The generation step implements the first only.  Allocation and compaction
 * accept any valid layout. */
diffkv_status diffkv_layout_init(diffkv_layout* out, int32_t head_dim, int32_t group,
                                 const int32_t k_bits[2], const int32_t v_bits[2],
                                 const int32_t tokens_per_page[2], int32_t max_seq_len);

enum {
    DIFFKV_OP_APPEND = 0,
    DIFFKV_OP_ATTENTION = 1,
    DIFFKV_OP_COMPACT = 2,
    DIFFKV_OP_ALLOC = 3,
    DIFFKV_OP_GENERATION = 4,
    DIFFKV_OP_PROMPT_SIGNIFICANCE = 5
};

/* Bytes of device workspace the operation needs (host out-parameter).
 * APPEND: num_seqs, num_kv_heads, total_new.  ATTENTION: num_seqs,
 * num_q_heads, num_splits (0 = automatic, -1 = balanced).
 * COMPACT / ALLOC / GENERATION: num_seqs*num_kv_heads tables.
 * PROMPT_SIGNIFICANCE: num_seqs, num_q_heads, total_new.  Unused sizes
 * are ignored. */
diffkv_status diffkv_workspace_size(int32_t op, const diffkv_layout* layout,
                                    int32_t num_seqs, int32_t num_q_heads,
                                    int32_t num_kv_heads, int64_t total_new,
                                    int32_t num_splits, size_t* bytes);

/*
 * KV compressor (Sec. 4) + page placement (Sec. 5.2, 5.3): classes the new
 * tokens of every table, reserves the pages both sections now need with one
 * prefix-sum schedule over all tables, then quantizes and stores every kept
 * token.
 *
 *   new_len  device int32 [num_seqs]: new tokens of sequence b; their rows in
 *            k/v/score are new_off(b) .. +new_len[b]-1, new_off(b) =
 *            sum of new_len[0..b).  Must sum to total_new with every entry in
 *            [0, max_new], else DIFFKV_ST_BAD_INPUT is raised and nothing
 *            changes.
 *   k, v     device fp16 [total_new][num_kv_heads][head_dim].
 *   score    device fp32 [total_new][num_kv_heads]: significance (not NaN).
 *   quota    device int32 [num_seqs][num_kv_heads][2] = {n_high, n_low}, or
 *            NULL.  Quota form: the non-window new tokens are ranked by
 *            (score descending, position ascending; -0 == +0); the first
 *            min(n_high, avail) are high, the next min(n_low, avail - n_high')
 *            low, the rest pruned.  Threshold form (quota == NULL; Sec. 4,
 *            Algorithm 1): high iff score >= alpha_h / N, else low iff
 *            score >= alpha_l / N, else pruned, N = seq_len[b] + new_len[b]
 *            and both thresholds computed in fp32.
 *   recent_window  the last W new tokens of each sequence are high precision
 *            and outside the quotas (W >= 0).
 *
 * Quantization (Sec. 2.2) per 32-dim group of each kept K and V vector:
 *   s = fp16_rne((max - min) / (2^b - 1)) in fp32, z = min (with -0 -> +0),
 *   code = clamp(rint((x - z) / s), 0, 2^b - 1) in fp32 with the stored fp16
 *   s and z, code = 0 when s == 0; b = k_bits/v_bits of the token's class.
 * Placement: kept tokens of a section take section indices len .. in
 *   position order.  Page demand per section = ceil((len + added) / T) -
 *   pages (if positive).  Tables take their new IDs from the ring region
 *   after the demands of all lower tables, high pages first; head advances
 *   by the total.  Raises OUT_OF_PAGES / TABLE_OVERFLOW all-or-nothing.
 * Updates pool, page_table, pages, len, seq_len (+= new_len), ring_ptr[0].
 * Workspace: diffkv_workspace_size(DIFFKV_OP_APPEND, ...); it needs no
 * clearing between calls.  A call with max_new <= 1 over at most 1024 tables
 * (a decode step) runs as one launch.
 */
diffkv_status diffkv_quantize_append(const diffkv_layout* layout, const diffkv_cache* cache,
                                     int64_t total_new, int32_t max_new,
                                     const int32_t* new_len,
                                     const uint16_t* k, const uint16_t* v,
                                     const float* score, const int32_t* quota,
                                     float alpha_h, float alpha_l, int32_t recent_window,
                                     void* ws, size_t ws_bytes, void* stream);

/*
 * Decode attention over the compressed cache, Eq. (1) of Sec. 2.1, one new
 * query per sequence and query head (Sec. 6.2):
 *   out[b][hq] = sum_j softmax_j(sm_scale * q[b][hq] . k_hat_j) v_hat_j
 * over every kept token of table b*Hkv + hq/(Hq/Hkv): the high section, then
 * the low section; k_hat = s*code + z per group.  fp32 accumulation.
 *   q    device fp16 [num_seqs][num_q_heads][head_dim]
 *   out  device fp32 [num_seqs][num_q_heads][head_dim]
 *   lse  device fp32 [num_seqs][num_q_heads] (natural log of the softmax
 *        denominator incl. the max) or NULL.  An empty table gives out = 0,
 *        lse = -inf.
 *   num_splits  0 = automatic (default): no table is split when there are
 *        at least as many tables as eight-wave workgroups the device holds at
 *        once -- up to 5 query heads per KV head each workgroup takes two
 *        tables (one long, one short: ranks j and T-1-j by decreasing work)
 *        and splits its waves between them by their work; above, one
 *        workgroup per table (waves with more pages left get issue priority)
 *        -- otherwise the balanced mode.
 *        -1 = balanced: the page lists of all tables, in table order, form one
 *        list of work units (a high page 3, a 32-token low page 6, a 16-token
 *        low page 3, a table's start 50) cut into one equal
 *        share per resident workgroup; a table spread over several shares has
 *        their (max, sum, acc) states merged in page order (Sec. 6.2 sequence
 *        split).  S >= 1: each table is cut into min(S, pages) equal page
 *        ranges, merged the same way (S = 1: no split, no merge).  Results
 *        are deterministic for a given mode and device.
 *   ws   device workspace of diffkv_workspace_size(DIFFKV_OP_ATTENTION, ...)
 *        bytes (always needed: it holds the split tables' partial states and
 *        one arrival word per table, which each call tags as its own, so the
 *        workspace needs no clearing between calls).
 * num_q_heads must be a multiple of num_kv_heads, with at most 8 query heads
 * per KV head.
 * Precision: q . k_hat is exact up to fp32 summation (codes and q enter fp16
 * products exactly); each value weight p * s_v is rounded to fp16 (relative
 * 2^-11, the rounding charged at the centre code), so an output differs from
 * exact Eq. (1) by at most about 2^-12 * R plus fp32 rounding, R being the
 * largest dequantized value-group range of its table.  Any finite fp16 cache
 * is accepted: the weights never overflow fp16 (pages with a value scale above
 * 2^7 keep them <= s_v).
 */
diffkv_status diffkv_decode_attention(const diffkv_layout* layout, const diffkv_cache* cache,
                                      int32_t num_q_heads, const uint16_t* q, float sm_scale,
                                      float* out, float* lse, int32_t num_splits,
                                      void* ws, size_t ws_bytes, void* stream);

/*
 * diffkv_decode_attention without a workspace, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc).  Same arguments, minus ws / ws_bytes, and
 * the same kernels and results, bit for bit.  The arrival words and split
 * partial states go to a fixed 8 MiB array in the library's device memory, one
 * per device, held from the library's load until the process ends; its device
 * address is looked up on the first call on each device and kept (the one
 * piece of state the library keeps).  A call whose mode, as resolved on the
 * current device, needs more -- the balanced mode takes 8 B per table plus
 * (resident workgroups + tables) * (Hq/Hkv) * 520 B -- returns
 * DIFFKV_E_SCRATCH and enqueues nothing.  Nothing in the scratch needs
 * clearing between calls.  Every call on a device shares that device's array:
 * calls ordered on one stream are safe, calls that may overlap on one device
 * (unordered streams) race.  Allocates, frees and synchronizes nothing.
 */
diffkv_status diffkv_decode_attention_noalloc(const diffkv_layout* layout, const diffkv_cache* cache,
                                              int32_t num_q_heads, const uint16_t* q, float sm_scale,
                                              float* out, float* lse, int32_t num_splits, void* stream);

/*
 * Significance update of one decode step (Sec. 4: a token's significance is
 * the average of the attention scores it receives; with grouped heads the
 * scores of a KV head's query heads are combined by their maximum).  Call it
 * after diffkv_decode_attention with the same q, passing that call's lse.
 * For every kept token j of table t = b*Hkv + h at position pos_j:
 *   x_j = max over the query heads hq of KV head h of exp(logit_hq,j - lse_hq),
 *         logit = sm_scale * q[b][hq] . k_hat_j (the probability of token j
 *         in the softmax over the table's kept tokens),
 *   score_j <- score_j + (x_j - score_j) / (N - pos_j),  N = seq_len[b],
 * i.e. the mean over the N - pos_j queries (positions pos_j .. N-1) the token
 * has received, the newest being this step's.  Scores are rewritten in place
 * in the pages' score segments; nothing else changes.  fp32 arithmetic.
 *   q    device fp16 [num_seqs][num_q_heads][head_dim] (as given to attention)
 *   lse  device fp32 [num_seqs][num_q_heads] (natural log, as attention wrote it)
 * No workspace.  Same layout and group-size support as diffkv_decode_attention.
 */
diffkv_status diffkv_update_significance(const diffkv_layout* layout, const diffkv_cache* cache,
                                         int32_t num_q_heads, const uint16_t* q, float sm_scale,
                                         const float* lse, void* stream);

/*
 * Prompt-phase significance (Sec. 4): the score of every prompt token, from
 * the prompt's own queries and fp16 keys, before the prompt is appended.
 * For sequence b with N = new_len[b] prompt tokens and KV head h, token p
 * (0-based) gets
 *   score[p][h] = (1 / (N - p)) * sum_{j = p}^{N-1} max_{hq of h} P_hq[j][p],
 *   P_hq[j][.] = softmax over p' <= j of sm_scale * q[j][hq] . k[p'][h],
 * the mean of the N - p causal attention probabilities the token receives,
 * the KV head's query heads combined by their maximum per query (the score
 * diffkv_update_significance continues).  The result feeds the `score`
 * argument of diffkv_quantize_append directly (same rows, same order).
 *   new_len  device int32 [num_seqs]; rows of sequence b follow those of b-1.
 *            Lengths are clamped to [0, max_new] and rows past total_new are
 *            neither read nor scored.
 *   q        device fp16 [total_new][num_q_heads][128], 16-byte aligned
 *   k        device fp16 [total_new][num_kv_heads][128], 16-byte aligned
 *   lse      device fp32 [total_new][num_q_heads] natural-log row normalizers
 *            (as a prompt attention kernel writes them), or NULL: the call
 *            computes them in an extra pass over q and k.
 *   score    device fp32 [total_new][num_kv_heads] out
 *   ws       diffkv_workspace_size(DIFFKV_OP_PROMPT_SIGNIFICANCE, ...) bytes
 * Arithmetic: fp16 x fp16 products on the matrix cores (exact), fp32 sums,
 * fp32 softmax with exp2; probabilities below 2^-126 may come out as zero.
 * sm_scale must be positive and finite (DIFFKV_E_INVAL otherwise).
 * num_q_heads / num_kv_heads up to 8 (else DIFFKV_E_UNSUPPORTED).
 */
diffkv_status diffkv_prompt_significance(const diffkv_layout* layout, int32_t num_seqs, int64_t total_new,
                                         int32_t max_new, const int32_t* new_len, int32_t num_q_heads,
                                         int32_t num_kv_heads, const uint16_t* q, const uint16_t* k,
                                         float sm_scale, const float* lse, float* score, void* ws,
                                         size_t ws_bytes, void* stream);

/*
 * Parallel free-list compaction (Sec. 5.2 recycling, Sec. 5.3): for the
 * first num_tables tables, every live slot whose release byte is nonzero
 * gives its page back.  With one prefix sum over tables, table t writes its
 * released IDs -- in ascending slot order -- to ring[(tail + off_t + i) % n];
 * tail advances by the total.  Each table is then squeezed in place: kept
 * high IDs packed from slot 0 and kept low IDs from slot p_max-1, both in
 * their section order; vacated slots become -1.  A released page removes its
 * tokens from the section (T, or the tail page's fill; later pages shift
 * down).  Request completion = releasing every live slot of its tables.
 *   release  device uint8 [num_tables][p_max]; bytes of non-live slots are
 *            ignored.
 * Never fails on the device (released IDs always fit the ring).  p_max above
 * 8192 or more than 2^20 tables: DIFFKV_E_UNSUPPORTED.
 */
diffkv_status diffkv_compact_free_list(const diffkv_layout* layout, const diffkv_cache* cache,
                                       int32_t num_tables, const uint8_t* release,
                                       void* ws, size_t ws_bytes, void* stream);

/*
 * Page allocation alone (Sec. 5.2 allocation; the prompt phase's
 * conservative reservation of Sec. 5.3): table t appends demand[t][HIGH]
 * pages to its high side and demand[t][LOW] to its low side, reading IDs
 * from the ring region after the demands of tables 0..t-1; head advances by
 * the total.  len is unchanged (the new pages are spare until an append
 * fills them).  All-or-nothing OUT_OF_PAGES / TABLE_OVERFLOW.
 *   demand  device int32 [num_tables][2], entries >= 0.
 */
diffkv_status diffkv_alloc_pages(const diffkv_layout* layout, const diffkv_cache* cache,
                                 int32_t num_tables, const int32_t* demand,
                                 void* ws, size_t ws_bytes, void* stream);

/*
 * Generation-phase policy (Sec. 4, Algorithm 1), once per decode step, after
 * the step's diffkv_quantize_append has put the newest token of every
 * sequence into the high section (its recent window).  For table t of
 * sequence b, with N = seq_len[b] and W = recent_window:
 *   - candidate: the high token at position N - 1 - W (the one that has just
 *     left the window); a table without one is left alone;
 *   - thresholds alpha_h / N and alpha_l / N, fp32 quotients;
 *   - victim of a section: its token of lowest score (-0 == +0; ties to the
 *     lowest position) among those at positions <= N - 1 - W;
 *   - score(candidate) >= alpha_h/N: the candidate stays; the high victim
 *     moves to the low section if alpha_l/N <= its score < alpha_h/N, and is
 *     removed if its score < alpha_l/N;
 *   - alpha_l/N <= score(candidate) < alpha_h/N: the candidate moves to the
 *     low section, over the low victim's slot if that victim's score is
 *     < alpha_l/N (the victim is evicted), else at the section's end;
 *   - otherwise the candidate is removed.
 * A token leaves the high section by swap-remove: the section's last token
 * moves into its slot (bytes unchanged) and the vacated slot is cleared to
 * zero; a page emptied this way stays with the table.  A token moving to the
 * low section is re-quantized: per element s*code + z as one fp32 fma,
 * rounded to fp16 (nearest even), then quantized as diffkv_quantize_append
 * quantizes a low-precision token; its score and position are kept.
 * Appending to a full low section takes one page per table, with the
 * allocation's prefix-sum schedule over tables (ring region after the pages
 * of lower tables; head advances by the total); all-or-nothing
 * OUT_OF_PAGES / TABLE_OVERFLOW (then nothing changes).  seq_len is not
 * changed.  Sections are dense but, after a removal, no longer in position
 * order (attention does not depend on the order).
 *   recent_window  W >= 0, DIFFKV_E_INVAL otherwise.
 *   ws   device workspace of diffkv_workspace_size(DIFFKV_OP_GENERATION, ...).
 */
diffkv_status diffkv_generation_step(const diffkv_layout* layout, const diffkv_cache* cache,
                                     float alpha_h, float alpha_l, int32_t recent_window,
                                     void* ws, size_t ws_bytes, void* stream);

/* Static string for a diffkv_status value. */
const char* diffkv_status_str(diffkv_status s);

#ifdef __cplusplus
}
#endif
#endif
