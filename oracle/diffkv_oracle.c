/*
 * diffkv_oracle.c -- serial CPU reference of the DiffKV hot path.
 * TEST INFRASTRUCTURE ONLY (see diffkv_oracle.h).  Plain C11, fp64 where the
 * paper leaves the precision open, IEEE fp32 where the quantizer must agree
 * bit for bit with the GPU.  Build: gcc -O2 -ffp-contract=off -fPIC -shared.
 */
#include "diffkv_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>

/* ======================================================================
 * fp16 <-> fp32 (IEEE 754 binary16), by bit manipulation.
 * ====================================================================== */
float dko_half_to_float(uint16_t h)
{
    uint32_t sign = (uint32_t)(h & 0x8000u) << 16;
    uint32_t exp = (h >> 10) & 0x1fu;
    uint32_t man = h & 0x3ffu;
    uint32_t bits;
    if (exp == 0) {
        if (man == 0) {
            bits = sign;
        } else { /* subnormal: man * 2^-24, renormalise */
            int e = -1;
            do { man <<= 1; e++; } while ((man & 0x400u) == 0);
            man &= 0x3ffu;
            bits = sign | ((uint32_t)(127 - 15 - e) << 23) | (man << 13);
        }
    } else if (exp == 31) {
        bits = sign | 0x7f800000u | (man << 13);
    } else {
        bits = sign | ((exp - 15 + 127) << 23) | (man << 13);
    }
    float f;
    memcpy(&f, &bits, 4);
    return f;
}

/* round to nearest, ties to even */
static uint32_t rne_shift(uint32_t m, int sh)
{
    if (sh <= 0) return m;
    if (sh >= 32) return 0;
    uint32_t q = m >> sh;
    uint32_t rem = m & ((1u << sh) - 1u);
    uint32_t half = 1u << (sh - 1);
    if (rem > half || (rem == half && (q & 1u))) q++;
    return q;
}

uint16_t dko_float_to_half(float f)
{
    uint32_t x;
    memcpy(&x, &f, 4);
    uint16_t sign = (uint16_t)((x >> 16) & 0x8000u);
    uint32_t ax = x & 0x7fffffffu;
    if (ax >= 0x7f800000u) { /* inf / nan */
        if (ax > 0x7f800000u) return (uint16_t)(sign | 0x7e00u | ((ax >> 13) & 0x3ffu));
        return (uint16_t)(sign | 0x7c00u);
    }
    if (ax >= 0x477ff000u) return (uint16_t)(sign | 0x7c00u); /* >= 65520 */
    if (ax < 0x33000000u) return sign;                         /* < 2^-25 */
    uint32_t e = ax >> 23;
    uint32_t m = (ax & 0x7fffffu) | 0x800000u;
    if (ax < 0x38800000u) { /* result is subnormal: units of 2^-24 */
        int sh = 126 - (int)e;
        return (uint16_t)(sign | rne_shift(m, sh));
    }
    /* normal: 10 kept mantissa bits, carry may bump the exponent */
    uint32_t q = ((e - 112u) << 10) | ((ax & 0x7fffffu) >> 13);
    uint32_t rem = ax & 0x1fffu;
    if (rem > 0x1000u || (rem == 0x1000u && (q & 1u))) q++;
    return (uint16_t)(sign | q);
}

void dko_half_to_float_n(int64_t n, const uint16_t* h, float* f)
{
    for (int64_t i = 0; i < n; i++) f[i] = dko_half_to_float(h[i]);
}

void dko_float_to_half_n(int64_t n, const float* f, uint16_t* h)
{
    for (int64_t i = 0; i < n; i++) h[i] = dko_float_to_half(f[i]);
}

/* ======================================================================
 * Quantization of one group (Sec. 2.2): scale and zero-point from the
 * group's min and max, codes round((x - z) / s), both kept as fp16.
 * Readings: s = (max - min) / (2^b - 1), z = min; the stored fp16 values
 * are the ones the codes are computed with; round half to even; codes
 * clamped to [0, 2^b - 1]; s == 0 gives all-zero codes; -0 counts as +0.
 * ====================================================================== */
void dko_quantize_group(const uint16_t* x, int n, int bits,
                        uint16_t* scale, uint16_t* zero, uint8_t* codes)
{
    float vals[256];
    int lb = (1 << bits) - 1;
    if (n <= 0 || n > 256) return;
    for (int i = 0; i < n; i++) vals[i] = dko_half_to_float(x[i]) + 0.0f;
    float mn = vals[0], mx = vals[0];
    for (int i = 1; i < n; i++) {
        if (vals[i] < mn) mn = vals[i];
        if (vals[i] > mx) mx = vals[i];
    }
    float s32 = (mx - mn) / (float)lb;
    uint16_t s16 = dko_float_to_half(s32);
    uint16_t z16 = dko_float_to_half(mn);
    float s = dko_half_to_float(s16);
    float z = dko_half_to_float(z16);
    for (int i = 0; i < n; i++) {
        if (s16 == 0) {
            codes[i] = 0;
            continue;
        }
        float r = rintf((vals[i] - z) / s);
        if (r < 0.0f) r = 0.0f;
        if (r > (float)lb) r = (float)lb;
        codes[i] = (uint8_t)r;
    }
    *scale = s16;
    *zero = z16;
}

/* ======================================================================
 * Layout of a unified page (Sec. 5.2): six segments in this order, each
 * starting on a 64-byte boundary:
 *   K codes  [D*kb/128 chunks][T][16 bytes]; chunk c holds dims
 *            c*(128/kb) .. +128/kb-1 of one token, element e at bit e*kb
 *   K meta   [T][D/G] {fp16 scale, fp16 zero}
 *   V codes  [D][T*vb/8 bytes]; token slot s of dim d at bit s*vb
 *   V meta   [D/G][T] {fp16 scale, fp16 zero}
 *   score    [T] fp32
 *   position [T] int32
 * Bits are little-endian within bytes, bytes little-endian within words.
 * Page stride = the larger of the two precisions' sizes (64-byte rounded).
 * Table width p_max = ceil(max_seq_len / T_high) + 1.
 * ====================================================================== */
static int32_t align64(int64_t x) { return (int32_t)((x + 63) & ~(int64_t)63); }

static int valid_bits(int b) { return b == 1 || b == 2 || b == 4 || b == 8; }

int dko_layout_init(dko_layout* L, int head_dim, int group,
                    const int32_t k_bits[2], const int32_t v_bits[2],
                    const int32_t tokens_per_page[2], int max_seq_len)
{
    memset(L, 0, sizeof(*L));
    if (head_dim <= 0 || group <= 0 || head_dim % group != 0 || group > 256) return 1;
    if (max_seq_len <= 0) return 1;
    for (int p = 0; p < 2; p++) {
        if (!valid_bits(k_bits[p]) || !valid_bits(v_bits[p])) return 1;
        if (tokens_per_page[p] <= 0) return 1;
        if ((head_dim * k_bits[p]) % 128 != 0) return 1;
        if ((tokens_per_page[p] * v_bits[p]) % 8 != 0) return 1;
    }
    if (tokens_per_page[1] < tokens_per_page[0]) return 1;
    L->head_dim = head_dim;
    L->group = group;
    L->max_seq_len = max_seq_len;
    int ng = head_dim / group;
    int64_t page = 0;
    for (int p = 0; p < 2; p++) {
        int T = tokens_per_page[p];
        L->k_bits[p] = k_bits[p];
        L->v_bits[p] = v_bits[p];
        L->tokens_per_page[p] = T;
        int64_t off = 0;
        L->off_kcode[p] = (int32_t)off; off = align64(off + (int64_t)(head_dim * k_bits[p] / 128) * T * 16);
        L->off_kmeta[p] = (int32_t)off; off = align64(off + (int64_t)T * ng * 4);
        L->off_vcode[p] = (int32_t)off; off = align64(off + (int64_t)head_dim * (T * v_bits[p] / 8));
        L->off_vmeta[p] = (int32_t)off; off = align64(off + (int64_t)ng * T * 4);
        L->off_score[p] = (int32_t)off; off = align64(off + (int64_t)T * 4);
        L->off_pos[p] = (int32_t)off;   off = align64(off + (int64_t)T * 4);
        L->used_bytes[p] = (int32_t)off;
        if (off > page) page = off;
    }
    L->page_bytes = page;
    L->p_max = (max_seq_len + tokens_per_page[0] - 1) / tokens_per_page[0] + 1;
    return 0;
}

/* ======================================================================
 * Classing (Sec. 4).  Quota form: rank the non-window tokens by
 * (score descending, position ascending); the first n_hi are high
 * precision, the next n_lo low precision, the rest pruned.  Threshold
 * form (Algorithm 1 comparisons): high iff score >= alpha_h / N, else low
 * iff score >= alpha_l / N, else pruned; N = sequence length after the
 * append, thresholds computed in fp32.
 * ====================================================================== */
typedef struct { float s; int j; } dko_key;

static int key_cmp(const void* a, const void* b)
{
    const dko_key* x = (const dko_key*)a;
    const dko_key* y = (const dko_key*)b;
    if (x->s > y->s) return -1;
    if (x->s < y->s) return 1;
    return (x->j < y->j) ? -1 : (x->j > y->j);
}

void dko_classify(int n, const float* score, const int32_t* quota,
                  float alpha_h, float alpha_l, int seq_len_after,
                  int window, int8_t* cls)
{
    int w = window < 0 ? 0 : (window > n ? n : window);
    int avail = n - w;
    for (int j = avail; j < n; j++) cls[j] = DKO_HIGH;
    if (avail <= 0) return;
    if (quota) {
        int nh = quota[0] < 0 ? 0 : quota[0];
        int nl = quota[1] < 0 ? 0 : quota[1];
        if (nh > avail) nh = avail;
        if (nl > avail - nh) nl = avail - nh;
        dko_key* keys = (dko_key*)malloc(sizeof(dko_key) * (size_t)avail);
        for (int j = 0; j < avail; j++) { keys[j].s = score[j]; keys[j].j = j; }
        qsort(keys, (size_t)avail, sizeof(dko_key), key_cmp);
        for (int r = 0; r < avail; r++) {
            int8_t c = (r < nh) ? DKO_HIGH : (r < nh + nl ? DKO_LOW : DKO_CLASS_PRUNE);
            cls[keys[r].j] = c;
        }
        free(keys);
    } else {
        float thr_h = alpha_h / (float)seq_len_after;
        float thr_l = alpha_l / (float)seq_len_after;
        for (int j = 0; j < avail; j++) {
            float s = score[j];
            cls[j] = (s >= thr_h) ? DKO_HIGH : (s >= thr_l ? DKO_LOW : DKO_CLASS_PRUNE);
        }
    }
}

/* ======================================================================
 * Allocation from the circular free page list (Sec. 5.2).  The demands of
 * all tables form one schedule: table t reads its page IDs from the ring
 * region that follows the demands of tables 0..t-1 (exclusive prefix sum),
 * high pages first (left side of the bidirectional table, left to right),
 * then low pages (right side, right to left).  All-or-nothing: if the
 * total exceeds the free region, or a table would hold more than p_max
 * pages, the status bit is set and nothing changes.
 * ====================================================================== */
static int alloc_core(const dko_layout* L, dko_cache* C, int num_tables,
                      const int32_t* need /* [num_tables][2] */)
{
    int64_t total = 0;
    uint32_t bad = 0;
    for (int t = 0; t < num_tables; t++) {
        int64_t nh = need[2 * t], nl = need[2 * t + 1];
        total += nh + nl;
        if ((int64_t)C->pages[2 * t] + nh + C->pages[2 * t + 1] + nl > L->p_max)
            bad |= DKO_ST_TABLE_OVERFLOW;
    }
    if (total > C->ring_ptr[1] - C->ring_ptr[0]) bad |= DKO_ST_OUT_OF_PAGES;
    if (bad) {
        *C->status |= bad;
        return 1;
    }
    int64_t head = C->ring_ptr[0];
    for (int t = 0; t < num_tables; t++) {
        int32_t* row = C->table + (int64_t)t * L->p_max;
        for (int i = 0; i < need[2 * t]; i++) {
            row[C->pages[2 * t]++] = C->ring[head % C->num_pages];
            head++;
        }
        for (int i = 0; i < need[2 * t + 1]; i++) {
            row[L->p_max - 1 - C->pages[2 * t + 1]++] = C->ring[head % C->num_pages];
            head++;
        }
    }
    C->ring_ptr[0] = head;
    return 0;
}

int dko_alloc_pages(const dko_layout* L, dko_cache* C, int num_tables,
                    const int32_t* demand)
{
    for (int i = 0; i < 2 * num_tables; i++)
        if (demand[i] < 0) return 1;
    alloc_core(L, C, num_tables, demand);
    return 0;
}

/* ======================================================================
 * Page access.
 * ====================================================================== */
static uint8_t* page_ptr(const dko_layout* L, const dko_cache* C, int t, int sec, int u)
{
    const int32_t* row = C->table + (int64_t)t * L->p_max;
    int T = L->tokens_per_page[sec];
    int pi = u / T;
    int32_t id = (sec == DKO_HIGH) ? row[pi] : row[L->p_max - 1 - pi];
    return C->pool + (int64_t)id * L->page_bytes;
}

static void put_bits(uint8_t* base, int64_t bit, int width, unsigned v)
{
    base[bit >> 3] |= (uint8_t)(v << (bit & 7));
    (void)width;
}

static unsigned get_bits(const uint8_t* base, int64_t bit, int width)
{
    return (base[bit >> 3] >> (bit & 7)) & ((1u << width) - 1u);
}

static void put_u16(uint8_t* p, uint16_t v) { p[0] = (uint8_t)v; p[1] = (uint8_t)(v >> 8); }
static uint16_t get_u16(const uint8_t* p) { return (uint16_t)(p[0] | (p[1] << 8)); }

/* Write one token (already classed into `sec`) into slot `slot` of page pg.
 * The slot's bytes are zero (fresh pages are cleared on their first slot). */
static void write_token(const dko_layout* L, uint8_t* pg, int sec, int slot,
                        const uint16_t* kvec, const uint16_t* vvec,
                        float score, int32_t pos)
{
    int D = L->head_dim, G = L->group, ng = D / G;
    int T = L->tokens_per_page[sec];
    int kb = L->k_bits[sec], vb = L->v_bits[sec];
    int per_chunk = 128 / kb;
    uint8_t codes[256];
    uint16_t s16, z16;
    for (int g = 0; g < ng; g++) {
        dko_quantize_group(kvec + g * G, G, kb, &s16, &z16, codes);
        for (int i = 0; i < G; i++) {
            int d = g * G + i;
            int c = d / per_chunk, e = d % per_chunk;
            uint8_t* chunk = pg + L->off_kcode[sec] + ((int64_t)c * T + slot) * 16;
            put_bits(chunk, (int64_t)e * kb, kb, codes[i]);
        }
        uint8_t* km = pg + L->off_kmeta[sec] + ((int64_t)slot * ng + g) * 4;
        put_u16(km, s16);
        put_u16(km + 2, z16);

        dko_quantize_group(vvec + g * G, G, vb, &s16, &z16, codes);
        int row_bytes = T * vb / 8;
        for (int i = 0; i < G; i++) {
            int d = g * G + i;
            uint8_t* row = pg + L->off_vcode[sec] + (int64_t)d * row_bytes;
            put_bits(row, (int64_t)slot * vb, vb, codes[i]);
        }
        uint8_t* vm = pg + L->off_vmeta[sec] + ((int64_t)g * T + slot) * 4;
        put_u16(vm, s16);
        put_u16(vm + 2, z16);
    }
    memcpy(pg + L->off_score[sec] + slot * 4, &score, 4);
    memcpy(pg + L->off_pos[sec] + slot * 4, &pos, 4);
}

void dko_read_token(const dko_layout* L, const dko_cache* C, int t, int sec,
                    int u, double* k_hat, double* v_hat,
                    float* score, int32_t* pos)
{
    int D = L->head_dim, G = L->group, ng = D / G;
    int T = L->tokens_per_page[sec];
    int kb = L->k_bits[sec], vb = L->v_bits[sec];
    int per_chunk = 128 / kb;
    int slot = u % T;
    const uint8_t* pg = page_ptr(L, C, t, sec, u);
    for (int d = 0; d < D; d++) {
        int g = d / G;
        int c = d / per_chunk, e = d % per_chunk;
        const uint8_t* chunk = pg + L->off_kcode[sec] + ((int64_t)c * T + slot) * 16;
        unsigned code = get_bits(chunk, (int64_t)e * kb, kb);
        const uint8_t* km = pg + L->off_kmeta[sec] + ((int64_t)slot * ng + g) * 4;
        double s = dko_half_to_float(get_u16(km)), z = dko_half_to_float(get_u16(km + 2));
        if (k_hat) k_hat[d] = s * (double)code + z;

        int row_bytes = T * vb / 8;
        const uint8_t* row = pg + L->off_vcode[sec] + (int64_t)d * row_bytes;
        code = get_bits(row, (int64_t)slot * vb, vb);
        const uint8_t* vm = pg + L->off_vmeta[sec] + ((int64_t)g * T + slot) * 4;
        s = dko_half_to_float(get_u16(vm));
        z = dko_half_to_float(get_u16(vm + 2));
        if (v_hat) v_hat[d] = s * (double)code + z;
    }
    if (score) memcpy(score, pg + L->off_score[sec] + slot * 4, 4);
    if (pos) memcpy(pos, pg + L->off_pos[sec] + slot * 4, 4);
}

/* ======================================================================
 * Compressor + placement.  For each table (sequence b, KV head h): class
 * the new tokens, reserve the pages the two sections now need (one
 * schedule for all tables), then quantize every kept token into its
 * section at index u = old section length + rank among this call's kept
 * tokens of the section (positions ascending).  Token u of a section lives
 * in slot u mod T of the section's page u / T.
 * ====================================================================== */
int dko_quantize_append(const dko_layout* L, dko_cache* C,
                        const int32_t* new_len,
                        const uint16_t* k, const uint16_t* v,
                        const float* score, const int32_t* quota,
                        float alpha_h, float alpha_l, int window)
{
    int B = C->num_seqs, H = C->num_kv_heads, D = L->head_dim;
    int num_tables = B * H;
    int64_t* off = (int64_t*)malloc(sizeof(int64_t) * (size_t)(B + 1));
    off[0] = 0;
    for (int b = 0; b < B; b++) off[b + 1] = off[b] + new_len[b];
    int64_t rows = off[B];
    int8_t* cls = (int8_t*)malloc((size_t)(rows * H > 0 ? rows * H : 1));
    int32_t* need = (int32_t*)calloc((size_t)num_tables * 2, sizeof(int32_t));
    int32_t* add = (int32_t*)calloc((size_t)num_tables * 2, sizeof(int32_t));
    float* sc = (float*)malloc(sizeof(float) * (size_t)(rows > 0 ? rows : 1));

    for (int b = 0; b < B; b++) {
        int n = new_len[b];
        int N = C->seq_len[b] + n;
        for (int h = 0; h < H; h++) {
            int t = b * H + h;
            int8_t* c = cls + (off[b] * H) + (int64_t)h * n;
            for (int j = 0; j < n; j++) sc[j] = score[(off[b] + j) * H + h];
            dko_classify(n, sc, quota ? quota + 2 * t : NULL, alpha_h, alpha_l, N, window, c);
            for (int j = 0; j < n; j++)
                if (c[j] >= 0) add[2 * t + c[j]]++;
            for (int sec = 0; sec < 2; sec++) {
                int T = L->tokens_per_page[sec];
                int want = (C->len[2 * t + sec] + add[2 * t + sec] + T - 1) / T;
                int have = C->pages[2 * t + sec];
                need[2 * t + sec] = want > have ? want - have : 0;
            }
        }
    }

    if (alloc_core(L, C, num_tables, need) == 0) {
        for (int b = 0; b < B; b++) {
            int n = new_len[b];
            for (int h = 0; h < H; h++) {
                int t = b * H + h;
                const int8_t* c = cls + (off[b] * H) + (int64_t)h * n;
                int cnt[2] = {0, 0};
                for (int j = 0; j < n; j++) {
                    if (c[j] < 0) continue;
                    int sec = c[j];
                    int u = C->len[2 * t + sec] + cnt[sec]++;
                    int T = L->tokens_per_page[sec];
                    uint8_t* pg = page_ptr(L, C, t, sec, u);
                    if (u % T == 0) memset(pg, 0, (size_t)L->page_bytes);
                    int64_t r = off[b] + j;
                    write_token(L, pg, sec, u % T,
                                k + (r * H + h) * D, v + (r * H + h) * D,
                                score[r * H + h], C->seq_len[b] + j);
                }
                C->len[2 * t] += cnt[0];
                C->len[2 * t + 1] += cnt[1];
            }
            C->seq_len[b] += n;
        }
    }
    free(off); free(cls); free(need); free(add); free(sc);
    return 0;
}

/* ======================================================================
 * Free-list compaction (Sec. 5.2 recycling, Sec. 5.3).  Per table, the
 * released live slots, in ascending slot order, write their page IDs to
 * the ring region that follows the releases of tables 0..t-1, starting at
 * the end pointer (wrapping).  The table is then squeezed: kept high pages
 * packed to the left, kept low pages to the right, both in their section
 * order; vacated slots become -1.  Each released page takes its tokens out
 * of the section length (a full page, or the tail page's fill).
 * ====================================================================== */
int dko_compact(const dko_layout* L, dko_cache* C, int num_tables,
                const uint8_t* release)
{
    int P = L->p_max;
    int64_t tail = C->ring_ptr[1];
    int32_t* keep = (int32_t*)malloc(sizeof(int32_t) * (size_t)P);
    for (int t = 0; t < num_tables; t++) {
        int32_t* row = C->table + (int64_t)t * P;
        const uint8_t* rel = release + (int64_t)t * P;
        int ph = C->pages[2 * t], pl = C->pages[2 * t + 1];
        int lens[2] = {C->len[2 * t], C->len[2 * t + 1]};
        int dropped[2] = {0, 0};
        for (int slot = 0; slot < P; slot++) {
            int sec, k;
            if (slot < ph) { sec = DKO_HIGH; k = slot; }
            else if (slot >= P - pl) { sec = DKO_LOW; k = P - 1 - slot; }
            else continue;
            if (!rel[slot]) continue;
            C->ring[tail % C->num_pages] = row[slot];
            tail++;
            int T = L->tokens_per_page[sec];
            int fill = lens[sec] - k * T;
            if (fill < 0) fill = 0;
            if (fill > T) fill = T;
            dropped[sec] += fill;
        }
        /* squeeze the high side */
        int nk = 0;
        for (int k = 0; k < ph; k++)
            if (!rel[k]) keep[nk++] = row[k];
        for (int k = 0; k < ph; k++) row[k] = (k < nk) ? keep[k] : -1;
        int newph = nk;
        /* squeeze the low side (section order k = 0.. is slot P-1, P-2, ..) */
        nk = 0;
        for (int k = 0; k < pl; k++)
            if (!rel[P - 1 - k]) keep[nk++] = row[P - 1 - k];
        for (int k = 0; k < pl; k++) row[P - 1 - k] = (k < nk) ? keep[k] : -1;
        C->pages[2 * t] = newph;
        C->pages[2 * t + 1] = nk;
        C->len[2 * t] -= dropped[0];
        C->len[2 * t + 1] -= dropped[1];
    }
    C->ring_ptr[1] = tail;
    free(keep);
    return 0;
}

/* ======================================================================
 * Generation phase (Sec. 4, Algorithm 1), once per decode step, after the
 * step's append has put the newest token into the high section as part of
 * the recent window.  Table t of sequence b, N = seq_len[b]:
 *   - the candidate t_c is the high token at position N - 1 - W, the one
 *     that has just left the window of the W most recent positions; a
 *     table without it is left alone;
 *   - thresholds alpha_h / N and alpha_l / N in fp32, as in the prompt
 *     phase; a victim is the token of lowest score (ties: lowest position)
 *     among a section's tokens outside the window (positions <= N - 1 - W);
 *   - score(t_c) >= alpha_h/N: t_c stays high; the high victim v moves to
 *     the low section if alpha_l/N <= score(v) < alpha_h/N and is removed
 *     if score(v) < alpha_l/N;
 *   - alpha_l/N <= score(t_c) < alpha_h/N: t_c moves to the low section;
 *     the low victim v is removed if score(v) < alpha_l/N (t_c, whose score
 *     is >= alpha_l/N, cannot be that victim, so t_c takes v's slot);
 *   - otherwise t_c is removed.
 * Removal keeps a section dense: its last token moves into the hole (raw
 * bytes) and the vacated slot is cleared; a page emptied this way stays with
 * the table.  A token entering the low section otherwise goes to its end;
 * the step takes a new page only then, from the ring with the append's
 * prefix-sum schedule (all-or-nothing).  Moving a token to the low section
 * re-quantizes it: each element dequantized as fmaf(s, code, z) in fp32,
 * rounded to fp16 (RNE), then quantized at the low precision exactly as an
 * append quantizes a new token.
 * ====================================================================== */
static void token_loc(const dko_layout* L, const dko_cache* C, int t, int sec, int u,
                      uint8_t** pg, int* slot)
{
    *pg = page_ptr(L, C, t, sec, u);
    *slot = u % L->tokens_per_page[sec];
}

static float token_score(const dko_layout* L, const dko_cache* C, int t, int sec, int u)
{
    uint8_t* pg;
    int slot;
    float s;
    token_loc(L, C, t, sec, u, &pg, &slot);
    memcpy(&s, pg + L->off_score[sec] + slot * 4, 4);
    return s;
}

static int32_t token_pos(const dko_layout* L, const dko_cache* C, int t, int sec, int u)
{
    uint8_t* pg;
    int slot;
    int32_t p;
    token_loc(L, C, t, sec, u, &pg, &slot);
    memcpy(&p, pg + L->off_pos[sec] + slot * 4, 4);
    return p;
}

/* Zero every bit of one slot (codes, metadata, score, position). */
static void clear_slot(const dko_layout* L, uint8_t* pg, int sec, int slot)
{
    int D = L->head_dim, ng = D / L->group, T = L->tokens_per_page[sec];
    int kb = L->k_bits[sec], vb = L->v_bits[sec];
    int chunks = D * kb / 128, row_bytes = T * vb / 8;
    for (int c = 0; c < chunks; c++) memset(pg + L->off_kcode[sec] + ((int64_t)c * T + slot) * 16, 0, 16);
    memset(pg + L->off_kmeta[sec] + (int64_t)slot * ng * 4, 0, (size_t)ng * 4);
    for (int d = 0; d < D; d++) {
        uint8_t* row = pg + L->off_vcode[sec] + (int64_t)d * row_bytes;
        int64_t bit = (int64_t)slot * vb;
        row[bit >> 3] &= (uint8_t)~(((1u << vb) - 1u) << (bit & 7));
    }
    for (int g = 0; g < ng; g++) memset(pg + L->off_vmeta[sec] + ((int64_t)g * T + slot) * 4, 0, 4);
    memset(pg + L->off_score[sec] + slot * 4, 0, 4);
    memset(pg + L->off_pos[sec] + slot * 4, 0, 4);
}

/* Copy token (sp, ss) to the cleared slot (dp, ds) of the same section. */
static void copy_slot(const dko_layout* L, const uint8_t* sp, int ss, uint8_t* dp, int ds, int sec)
{
    int D = L->head_dim, ng = D / L->group, T = L->tokens_per_page[sec];
    int kb = L->k_bits[sec], vb = L->v_bits[sec];
    int chunks = D * kb / 128, row_bytes = T * vb / 8;
    for (int c = 0; c < chunks; c++)
        memcpy(dp + L->off_kcode[sec] + ((int64_t)c * T + ds) * 16,
               sp + L->off_kcode[sec] + ((int64_t)c * T + ss) * 16, 16);
    memcpy(dp + L->off_kmeta[sec] + (int64_t)ds * ng * 4, sp + L->off_kmeta[sec] + (int64_t)ss * ng * 4,
           (size_t)ng * 4);
    for (int d = 0; d < D; d++) {
        unsigned code = get_bits(sp + L->off_vcode[sec] + (int64_t)d * row_bytes, (int64_t)ss * vb, vb);
        put_bits(dp + L->off_vcode[sec] + (int64_t)d * row_bytes, (int64_t)ds * vb, vb, code);
    }
    for (int g = 0; g < ng; g++)
        memcpy(dp + L->off_vmeta[sec] + ((int64_t)g * T + ds) * 4, sp + L->off_vmeta[sec] + ((int64_t)g * T + ss) * 4, 4);
    memcpy(dp + L->off_score[sec] + ds * 4, sp + L->off_score[sec] + ss * 4, 4);
    memcpy(dp + L->off_pos[sec] + ds * 4, sp + L->off_pos[sec] + ss * 4, 4);
}

/* Remove token u of a section: the last token takes its slot. */
static void remove_token(const dko_layout* L, dko_cache* C, int t, int sec, int u)
{
    int last = C->len[2 * t + sec] - 1;
    uint8_t *dp, *lp;
    int ds, ls;
    token_loc(L, C, t, sec, u, &dp, &ds);
    token_loc(L, C, t, sec, last, &lp, &ls);
    if (u != last) {
        clear_slot(L, dp, sec, ds);
        copy_slot(L, lp, ls, dp, ds, sec);
    }
    clear_slot(L, lp, sec, ls);
    C->len[2 * t + sec] = last;
}

/* Fp16 key and value of high token u, dequantized in fp32 (fmaf) and
 * rounded to fp16. */
static void requant_source(const dko_layout* L, const dko_cache* C, int t, int u,
                           uint16_t* k16, uint16_t* v16, float* score, int32_t* pos)
{
    int sec = DKO_HIGH;
    int D = L->head_dim, G = L->group, ng = D / G, T = L->tokens_per_page[sec];
    int kb = L->k_bits[sec], vb = L->v_bits[sec];
    int per_chunk = 128 / kb, row_bytes = T * vb / 8;
    uint8_t* pg;
    int slot;
    token_loc(L, C, t, sec, u, &pg, &slot);
    for (int d = 0; d < D; d++) {
        int g = d / G, c = d / per_chunk, e = d % per_chunk;
        unsigned code = get_bits(pg + L->off_kcode[sec] + ((int64_t)c * T + slot) * 16, (int64_t)e * kb, kb);
        const uint8_t* km = pg + L->off_kmeta[sec] + ((int64_t)slot * ng + g) * 4;
        k16[d] = dko_float_to_half(fmaf(dko_half_to_float(get_u16(km)), (float)code,
                                        dko_half_to_float(get_u16(km + 2))));
        code = get_bits(pg + L->off_vcode[sec] + (int64_t)d * row_bytes, (int64_t)slot * vb, vb);
        const uint8_t* vm = pg + L->off_vmeta[sec] + ((int64_t)g * T + slot) * 4;
        v16[d] = dko_float_to_half(fmaf(dko_half_to_float(get_u16(vm)), (float)code,
                                        dko_half_to_float(get_u16(vm + 2))));
    }
    memcpy(score, pg + L->off_score[sec] + slot * 4, 4);
    memcpy(pos, pg + L->off_pos[sec] + slot * 4, 4);
}

/* Write a re-quantized token into low slot u (its slot cleared first; the
 * first slot of a page clears the page, as an append does). */
static void put_low(const dko_layout* L, dko_cache* C, int t, int u, const uint16_t* k16,
                    const uint16_t* v16, float score, int32_t pos)
{
    uint8_t* pg;
    int slot;
    token_loc(L, C, t, DKO_LOW, u, &pg, &slot);
    if (u == C->len[2 * t + 1] && slot == 0) memset(pg, 0, (size_t)L->page_bytes);
    else clear_slot(L, pg, DKO_LOW, slot);
    write_token(L, pg, DKO_LOW, slot, k16, v16, score, pos);
}

/* Victim of a section: lowest score, ties to the lowest position, among
 * tokens at positions <= pc.  Returns its index or -1. */
static int victim(const dko_layout* L, const dko_cache* C, int t, int sec, int32_t pc)
{
    int best = -1;
    float bs = 0.0f;
    int32_t bp = 0;
    for (int u = 0; u < C->len[2 * t + sec]; u++) {
        int32_t p = token_pos(L, C, t, sec, u);
        if (p > pc) continue;
        float s = token_score(L, C, t, sec, u);
        if (best < 0 || s < bs || (s == bs && p < bp)) {
            best = u;
            bs = s;
            bp = p;
        }
    }
    return best;
}

enum { GEN_NONE = 0, GEN_HIGH_VICTIM_TO_LOW, GEN_HIGH_VICTIM_OUT, GEN_CAND_TO_LOW, GEN_CAND_OUT };

int dko_generation_step(const dko_layout* L, dko_cache* C, float alpha_h, float alpha_l, int window)
{
    int B = C->num_seqs, H = C->num_kv_heads, D = L->head_dim;
    int num_tables = B * H;
    int* act = (int*)calloc((size_t)num_tables, sizeof(int));
    int* uc = (int*)calloc((size_t)num_tables, sizeof(int));   /* candidate's high index */
    int* uv = (int*)calloc((size_t)num_tables, sizeof(int));   /* victim's index         */
    int32_t* need = (int32_t*)calloc((size_t)num_tables * 2, sizeof(int32_t));
    uint16_t* k16 = (uint16_t*)malloc(sizeof(uint16_t) * (size_t)D);
    uint16_t* v16 = (uint16_t*)malloc(sizeof(uint16_t) * (size_t)D);
    int w = window < 0 ? 0 : window;

    /* decide every table's action on the state before the step */
    for (int t = 0; t < num_tables; t++) {
        int N = C->seq_len[t / H];
        int32_t pc = N - 1 - w;
        act[t] = GEN_NONE;
        if (pc < 0) continue;
        int c = -1;
        for (int u = 0; u < C->len[2 * t]; u++)
            if (token_pos(L, C, t, DKO_HIGH, u) == pc) { c = u; break; }
        if (c < 0) continue;
        float thr_h = alpha_h / (float)N, thr_l = alpha_l / (float)N;
        float sc = token_score(L, C, t, DKO_HIGH, c);
        uc[t] = c;
        if (sc >= thr_h) {
            int v = victim(L, C, t, DKO_HIGH, pc);
            float sv = token_score(L, C, t, DKO_HIGH, v);
            uv[t] = v;
            if (sv >= thr_l && sv < thr_h) act[t] = GEN_HIGH_VICTIM_TO_LOW;
            else if (sv < thr_l) act[t] = GEN_HIGH_VICTIM_OUT;
        } else if (sc >= thr_l) {
            int v = victim(L, C, t, DKO_LOW, pc);
            uv[t] = (v >= 0 && token_score(L, C, t, DKO_LOW, v) < thr_l) ? v : -1;
            act[t] = GEN_CAND_TO_LOW;
        } else {
            act[t] = GEN_CAND_OUT;
        }
        /* a token goes to the end of the low section: a new page if it is full */
        int grows = act[t] == GEN_HIGH_VICTIM_TO_LOW || (act[t] == GEN_CAND_TO_LOW && uv[t] < 0);
        int T = L->tokens_per_page[DKO_LOW];
        if (grows && C->len[2 * t + 1] + 1 > C->pages[2 * t + 1] * T) need[2 * t + 1] = 1;
    }

    if (alloc_core(L, C, num_tables, need) == 0) {
        for (int t = 0; t < num_tables; t++) {
            float sc;
            int32_t pos;
            switch (act[t]) {
            case GEN_HIGH_VICTIM_TO_LOW:
                requant_source(L, C, t, uv[t], k16, v16, &sc, &pos);
                remove_token(L, C, t, DKO_HIGH, uv[t]);
                put_low(L, C, t, C->len[2 * t + 1], k16, v16, sc, pos);
                C->len[2 * t + 1]++;
                break;
            case GEN_HIGH_VICTIM_OUT:
                remove_token(L, C, t, DKO_HIGH, uv[t]);
                break;
            case GEN_CAND_TO_LOW:
                requant_source(L, C, t, uc[t], k16, v16, &sc, &pos);
                remove_token(L, C, t, DKO_HIGH, uc[t]);
                if (uv[t] >= 0) {
                    put_low(L, C, t, uv[t], k16, v16, sc, pos);
                } else {
                    put_low(L, C, t, C->len[2 * t + 1], k16, v16, sc, pos);
                    C->len[2 * t + 1]++;
                }
                break;
            case GEN_CAND_OUT:
                remove_token(L, C, t, DKO_HIGH, uc[t]);
                break;
            default:
                break;
            }
        }
    }
    free(act); free(uc); free(uv); free(need); free(k16); free(v16);
    return 0;
}

/* ======================================================================
 * Attention, Eq. (1), in fp64 over the dequantized cache.
 * ====================================================================== */
static int table_tokens(const dko_cache* C, int t) { return C->len[2 * t] + C->len[2 * t + 1]; }

static void decode_table(const dko_layout* L, const dko_cache* C, int t,
                         double* K, double* V)
{
    int D = L->head_dim, n = 0;
    for (int sec = 0; sec < 2; sec++)
        for (int u = 0; u < C->len[2 * t + sec]; u++, n++)
            dko_read_token(L, C, t, sec, u, K + (int64_t)n * D, V + (int64_t)n * D, NULL, NULL);
}

static void decode_table_keys(const dko_layout* L, const dko_cache* C, int t, double* K)
{
    int D = L->head_dim, n = 0;
    for (int sec = 0; sec < 2; sec++)
        for (int u = 0; u < C->len[2 * t + sec]; u++, n++)
            dko_read_token(L, C, t, sec, u, K + (int64_t)n * D, NULL, NULL, NULL);
}

int dko_attention(const dko_layout* L, const dko_cache* C, int num_q_heads,
                  const uint16_t* q, double sm_scale, double* out, double* lse)
{
    int B = C->num_seqs, H = C->num_kv_heads, D = L->head_dim;
    if (H <= 0 || num_q_heads % H != 0) return 1;
    int g = num_q_heads / H;
    for (int b = 0; b < B; b++) {
        for (int h = 0; h < H; h++) {
            int t = b * H + h;
            int n = table_tokens(C, t);
            double* K = (double*)malloc(sizeof(double) * (size_t)(n > 0 ? n : 1) * D);
            double* V = (double*)malloc(sizeof(double) * (size_t)(n > 0 ? n : 1) * D);
            double* logit = (double*)malloc(sizeof(double) * (size_t)(n > 0 ? n : 1));
            decode_table(L, C, t, K, V);
            for (int hq = h * g; hq < (h + 1) * g; hq++) {
                const uint16_t* qv = q + ((int64_t)b * num_q_heads + hq) * D;
                double* o = out + ((int64_t)b * num_q_heads + hq) * D;
                double m = -INFINITY;
                for (int j = 0; j < n; j++) {
                    double dot = 0.0;
                    for (int d = 0; d < D; d++)
                        dot += (double)dko_half_to_float(qv[d]) * K[(int64_t)j * D + d];
                    logit[j] = sm_scale * dot;
                    if (logit[j] > m) m = logit[j];
                }
                double l = 0.0;
                for (int d = 0; d < D; d++) o[d] = 0.0;
                for (int j = 0; j < n; j++) {
                    double w = exp(logit[j] - m);
                    l += w;
                    for (int d = 0; d < D; d++) o[d] += w * V[(int64_t)j * D + d];
                }
                if (n > 0)
                    for (int d = 0; d < D; d++) o[d] /= l;
                if (lse) lse[(int64_t)b * num_q_heads + hq] = (n > 0) ? m + log(l) : -INFINITY;
            }
            free(K); free(V); free(logit);
        }
    }
    return 0;
}

void dko_attention_partial(const dko_layout* L, const dko_cache* C,
                           int num_q_heads, const uint16_t* q,
                           double sm_scale, int b, int hq, int p0, int p1,
                           double* m_out, double* l_out, double* acc)
{
    int H = C->num_kv_heads, D = L->head_dim;
    int g = num_q_heads / H;
    int t = b * H + hq / g;
    int ph = C->pages[2 * t];
    const uint16_t* qv = q + ((int64_t)b * num_q_heads + hq) * D;
    double* kh = (double*)malloc(sizeof(double) * (size_t)D);
    double* vh = (double*)malloc(sizeof(double) * (size_t)D);
    /* pass 1: max logit over the range; pass 2: weights and sums */
    double m = -INFINITY;
    for (int pass = 0; pass < 2; pass++) {
        double l = 0.0;
        if (pass == 1)
            for (int d = 0; d < D; d++) acc[d] = 0.0;
        for (int p = p0; p < p1; p++) {
            int sec = (p < ph) ? DKO_HIGH : DKO_LOW;
            int k = (p < ph) ? p : p - ph;
            int T = L->tokens_per_page[sec];
            int u0 = k * T, u1 = (k + 1) * T;
            if (u1 > C->len[2 * t + sec]) u1 = C->len[2 * t + sec];
            for (int u = u0; u < u1; u++) {
                dko_read_token(L, C, t, sec, u, kh, vh, NULL, NULL);
                double dot = 0.0;
                for (int d = 0; d < D; d++) dot += (double)dko_half_to_float(qv[d]) * kh[d];
                double lg = sm_scale * dot;
                if (pass == 0) {
                    if (lg > m) m = lg;
                } else {
                    double w = exp(lg - m);
                    l += w;
                    for (int d = 0; d < D; d++) acc[d] += w * vh[d];
                }
            }
        }
        if (pass == 1) *l_out = l;
    }
    *m_out = m;
    free(kh); free(vh);
}

void dko_merge_partials(int S, int D, const double* m, const double* l,
                        const double* acc, double* out, double* lse)
{
    double M = -INFINITY;
    for (int s = 0; s < S; s++)
        if (m[s] > M) M = m[s];
    for (int d = 0; d < D; d++) out[d] = 0.0;
    if (M == -INFINITY) {
        if (lse) *lse = -INFINITY;
        return;
    }
    double Ls = 0.0;
    for (int s = 0; s < S; s++) {
        if (m[s] == -INFINITY) continue;
        double f = exp(m[s] - M);
        Ls += l[s] * f;
        for (int d = 0; d < D; d++) out[d] += acc[(int64_t)s * D + d] * f;
    }
    for (int d = 0; d < D; d++) out[d] /= Ls;
    if (lse) *lse = M + log(Ls);
}

/* ======================================================================
 * Significance scores (Sec. 4).  A token's significance is the average of
 * the attention scores it receives from the queries at and after its
 * position; with grouped heads the scores of the KV head's query heads are
 * combined by their maximum, taken per query so that one running mean per
 * token holds it.  One decode step adds the step's query: every kept token's
 * probability under each of the g heads (softmax over the table's kept
 * tokens, fp64), its maximum x over the heads, and the running mean over the
 * N - p queries a token at position p has now received.
 * ====================================================================== */
static void token_score_ptr(const dko_layout* L, dko_cache* C, int t, int sec, int u, float** sp,
                            int32_t* pos)
{
    int T = L->tokens_per_page[sec];
    uint8_t* pg = (uint8_t*)page_ptr(L, C, t, sec, u);
    *sp = (float*)(pg + L->off_score[sec] + (u % T) * 4);
    memcpy(pos, pg + L->off_pos[sec] + (u % T) * 4, 4);
}

int dko_update_significance(const dko_layout* L, dko_cache* C, int num_q_heads,
                            const uint16_t* q, double sm_scale)
{
    int B = C->num_seqs, H = C->num_kv_heads, D = L->head_dim;
    if (H <= 0 || num_q_heads % H != 0) return 1;
    int g = num_q_heads / H;
    for (int b = 0; b < B; b++) {
        int N = C->seq_len[b];
        for (int h = 0; h < H; h++) {
            int t = b * H + h;
            int n = table_tokens(C, t);
            if (n == 0) continue;
            double* K = (double*)malloc(sizeof(double) * (size_t)n * D);
            double* logit = (double*)malloc(sizeof(double) * (size_t)n);
            double* x = (double*)malloc(sizeof(double) * (size_t)n);
            decode_table_keys(L, C, t, K);
            for (int j = 0; j < n; j++) x[j] = 0.0;
            for (int hq = h * g; hq < (h + 1) * g; hq++) {
                const uint16_t* qv = q + ((int64_t)b * num_q_heads + hq) * D;
                double m = -INFINITY;
                for (int j = 0; j < n; j++) {
                    double dot = 0.0;
                    for (int d = 0; d < D; d++) dot += (double)dko_half_to_float(qv[d]) * K[(int64_t)j * D + d];
                    logit[j] = sm_scale * dot;
                    if (logit[j] > m) m = logit[j];
                }
                double l = 0.0;
                for (int j = 0; j < n; j++) l += exp(logit[j] - m);
                for (int j = 0; j < n; j++) {
                    double pj = exp(logit[j] - m) / l;
                    if (pj > x[j]) x[j] = pj;
                }
            }
            int j = 0;
            for (int sec = 0; sec < 2; sec++) {
                for (int u = 0; u < C->len[2 * t + sec]; u++, j++) {
                    float* sp;
                    int32_t pos;
                    token_score_ptr(L, C, t, sec, u, &sp, &pos);
                    double s = (double)*sp;
                    *sp = (float)(s + (x[j] - s) / (double)(N - pos));
                }
            }
            free(K); free(logit); free(x);
        }
    }
    return 0;
}

/* ======================================================================
 * Prompt-phase significance (Sec. 4).  Over a prompt of N tokens every
 * query j attends causally to the keys 0..j with the full-precision (fp16)
 * keys; token p receives the N - p probabilities of the queries p..N-1.
 * Its significance is their average, each probability being the maximum
 * over the g query heads of its KV head (taken per query, the reading the
 * decode-time update continues).  fp64 throughout; rows of q, k and score
 * are the prompt tokens concatenated sequence after sequence.  `select`
 * ([B][Hkv], nonzero = compute) limits the work to some tables; the scores
 * of the others are left untouched.
 * ====================================================================== */
int dko_prompt_significance(int B, const int32_t* new_len, int num_q_heads, int num_kv_heads,
                            int D, const uint16_t* q, const uint16_t* k, double sm_scale,
                            const uint8_t* select, float* score)
{
    int H = num_kv_heads;
    if (H <= 0 || num_q_heads % H != 0 || D <= 0) return 1;
    int g = num_q_heads / H;
    int64_t row0 = 0;
    for (int b = 0; b < B; b++) {
        int N = new_len[b];
        if (N < 0) return 1;
        for (int h = 0; h < H; h++) {
            if (N == 0 || (select && !select[b * H + h])) continue;
            double* Kd = (double*)malloc(sizeof(double) * (size_t)N * D);
            double* logit = (double*)malloc(sizeof(double) * (size_t)N);
            double* x = (double*)malloc(sizeof(double) * (size_t)N);
            double* sum = (double*)calloc((size_t)N, sizeof(double));
            double* qd = (double*)malloc(sizeof(double) * (size_t)D);
            for (int p = 0; p < N; p++)
                for (int d = 0; d < D; d++)
                    Kd[(int64_t)p * D + d] = dko_half_to_float(k[((row0 + p) * H + h) * D + d]);
            for (int j = 0; j < N; j++) {          /* query j: keys 0..j */
                for (int p = 0; p <= j; p++) x[p] = 0.0;
                for (int hq = h * g; hq < (h + 1) * g; hq++) {
                    const uint16_t* qv = q + ((row0 + j) * num_q_heads + hq) * D;
                    for (int d = 0; d < D; d++) qd[d] = dko_half_to_float(qv[d]);
                    double m = -INFINITY;
                    for (int p = 0; p <= j; p++) {
                        double dot = 0.0;
                        for (int d = 0; d < D; d++) dot += qd[d] * Kd[(int64_t)p * D + d];
                        logit[p] = sm_scale * dot;
                        if (logit[p] > m) m = logit[p];
                    }
                    double l = 0.0;
                    for (int p = 0; p <= j; p++) l += exp(logit[p] - m);
                    for (int p = 0; p <= j; p++) {
                        double pr = exp(logit[p] - m) / l;
                        if (pr > x[p]) x[p] = pr;
                    }
                }
                for (int p = 0; p <= j; p++) sum[p] += x[p];
            }
            for (int p = 0; p < N; p++) score[(row0 + p) * H + h] = (float)(sum[p] / (double)(N - p));
            free(Kd); free(logit); free(x); free(sum); free(qd);
        }
        row0 += N;
    }
    return 0;
}

/* Prompt-phase significance of the last m tokens of one N-token prompt and
 * KV head h: the same definition restricted to tokens N-m..N-1, which only
 * the queries N-m..N-1 reach (each still normalized over its keys 0..j).
 * q, k point at the prompt's first row ([N][Hq][D], [N][Hkv][D]).
 * score_tail[i] is the score of token N-m+i, fp64. */
int dko_prompt_significance_tail(int N, int num_q_heads, int num_kv_heads, int D, const uint16_t* q,
                                 const uint16_t* k, double sm_scale, int h, int m, double* score_tail)
{
    int H = num_kv_heads;
    if (H <= 0 || num_q_heads % H != 0 || D <= 0 || h < 0 || h >= H || m < 0 || m > N) return 1;
    int g = num_q_heads / H;
    int p0 = N - m;
    double* Kd = (double*)malloc(sizeof(double) * (size_t)N * D);
    double* logit = (double*)malloc(sizeof(double) * (size_t)N);
    double* x = (double*)malloc(sizeof(double) * (size_t)N);
    double* qd = (double*)malloc(sizeof(double) * (size_t)D);
    for (int p = 0; p < N; p++)
        for (int d = 0; d < D; d++) Kd[(int64_t)p * D + d] = dko_half_to_float(k[((int64_t)p * H + h) * D + d]);
    for (int i = 0; i < m; i++) score_tail[i] = 0.0;
    for (int j = p0; j < N; j++) {
        for (int p = p0; p <= j; p++) x[p] = 0.0;
        for (int hq = h * g; hq < (h + 1) * g; hq++) {
            const uint16_t* qv = q + ((int64_t)j * num_q_heads + hq) * D;
            for (int d = 0; d < D; d++) qd[d] = dko_half_to_float(qv[d]);
            double mx = -INFINITY;
            for (int p = 0; p <= j; p++) {
                double dot = 0.0;
                for (int d = 0; d < D; d++) dot += qd[d] * Kd[(int64_t)p * D + d];
                logit[p] = sm_scale * dot;
                if (logit[p] > mx) mx = logit[p];
            }
            double l = 0.0;
            for (int p = 0; p <= j; p++) l += exp(logit[p] - mx);
            for (int p = p0; p <= j; p++) {
                double pr = exp(logit[p] - mx) / l;
                if (pr > x[p]) x[p] = pr;
            }
        }
        for (int p = p0; p <= j; p++) score_tail[p - p0] += x[p];
    }
    for (int p = p0; p < N; p++) score_tail[p - p0] /= (double)(N - p);
    free(Kd); free(logit); free(x); free(qd);
    return 0;
}

/* ======================================================================
 * Memory accounting against FP16 (Sec. 1, Fig. 1): bits of the kept
 * key/value codes over the bits of n_total FP16 keys/values.
 * ====================================================================== */
void dko_kv_bits_fraction(const dko_layout* L, int n_hi, int n_lo,
                          int n_total, double* k_frac, double* v_frac)
{
    double full = 16.0 * (double)n_total;
    *k_frac = ((double)n_hi * L->k_bits[0] + (double)n_lo * L->k_bits[1]) / full;
    *v_frac = ((double)n_hi * L->v_bits[0] + (double)n_lo * L->v_bits[1]) / full;
}
