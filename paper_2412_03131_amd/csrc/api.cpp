// api.cpp -- the C ABI of include/diffkv.h: argument checks, workspace
// carving and kernel dispatch.  No allocation, no synchronisation.
#include <string.h>

#include "internal.hpp"

using namespace dkv;

namespace {

int64_t align256(int64_t x) { return (x + 255) & ~(int64_t)255; }
int32_t align64(int64_t x) { return (int32_t)((x + 63) & ~(int64_t)63); }
bool bits_ok(int b) { return b == 1 || b == 2 || b == 4 || b == 8; }

diffkv_status fill_layout(diffkv_layout* L, int32_t head_dim, int32_t group, const int32_t kb[2],
                          const int32_t vb[2], const int32_t tp[2], int32_t max_seq_len)
{
    if (!L || !kb || !vb || !tp) return DIFFKV_E_INVAL;
    if (head_dim <= 0 || group <= 0 || head_dim % group != 0 || group > 256 || max_seq_len <= 0)
        return DIFFKV_E_INVAL;
    for (int p = 0; p < 2; ++p) {
        if (!bits_ok(kb[p]) || !bits_ok(vb[p]) || tp[p] <= 0) return DIFFKV_E_INVAL;
        if ((head_dim * kb[p]) % 128 != 0 || (tp[p] * vb[p]) % 8 != 0) return DIFFKV_E_INVAL;
    }
    if (tp[1] < tp[0]) return DIFFKV_E_INVAL;
    diffkv_layout o;
    memset(&o, 0, sizeof(o));
    o.head_dim = head_dim;
    o.group = group;
    o.max_seq_len = max_seq_len;
    const int ng = head_dim / group;
    int64_t page = 0;
    for (int p = 0; p < 2; ++p) {
        const int T = tp[p];
        o.k_bits[p] = kb[p];
        o.v_bits[p] = vb[p];
        o.tokens_per_page[p] = T;
        int64_t off = 0;
        o.off_kcode[p] = (int32_t)off;
        off = align64(off + (int64_t)(head_dim * kb[p] / 128) * T * 16);
        o.off_kmeta[p] = (int32_t)off;
        off = align64(off + (int64_t)T * ng * 4);
        o.off_vcode[p] = (int32_t)off;
        off = align64(off + (int64_t)head_dim * (T * vb[p] / 8));
        o.off_vmeta[p] = (int32_t)off;
        off = align64(off + (int64_t)ng * T * 4);
        o.off_score[p] = (int32_t)off;
        off = align64(off + (int64_t)T * 4);
        o.off_pos[p] = (int32_t)off;
        off = align64(off + (int64_t)T * 4);
        o.used_bytes[p] = (int32_t)off;
        if (off > page) page = off;
    }
    o.page_bytes = page;
    o.p_max = (max_seq_len + tp[0] - 1) / tp[0] + 1;
    *L = o;
    return DIFFKV_OK;
}

// A layout passed in must be one diffkv_layout_init produced.
bool layout_valid(const diffkv_layout* L)
{
    if (!L) return false;
    diffkv_layout r;
    if (fill_layout(&r, L->head_dim, L->group, L->k_bits, L->v_bits, L->tokens_per_page,
                    L->max_seq_len) != DIFFKV_OK)
        return false;
    return memcmp(&r, L, sizeof(r)) == 0;
}

// Index of the caller's layout among the ones the kernels implement
// (kLayoutFmts: head_dim 128, group 32, the section formats and the segment
// offsets diffkv_layout_init gives them), or -1.
int layout_index(const diffkv_layout* L)
{
    if (L->head_dim != kD || L->group != kG) return -1;
    for (int li = 0; li < kNumLayouts; ++li) {
        const KvFmt f[2] = {kLayoutFmts[li].hi, kLayoutFmts[li].lo};
        bool ok = L->page_bytes == layout_page_bytes(li);
        for (int p = 0; p < 2; ++p) {
            const SecOffsets o = sec_offsets(f[p]);
            ok = ok && L->k_bits[p] == f[p].kb && L->v_bits[p] == f[p].vb && L->tokens_per_page[p] == f[p].T &&
                 L->off_kcode[p] == o.kc && L->off_kmeta[p] == o.km && L->off_vcode[p] == o.vc &&
                 L->off_vmeta[p] == o.vm && L->off_score[p] == o.sc && L->off_pos[p] == o.pos;
        }
        if (ok) return li;
    }
    return -1;
}
bool layout_kernels_supported(const diffkv_layout* L) { return layout_index(L) >= 0; }

bool cache_valid(const diffkv_cache* c)
{
    return c && c->page_table && c->pages && c->len && c->ring && c->ring_ptr && c->status &&
           c->num_pages > 0 && c->num_pages <= INT32_MAX && c->num_seqs >= 0 && c->num_kv_heads > 0 &&
           (int64_t)c->num_seqs * c->num_kv_heads <= INT32_MAX;
}

void fill_layout_args(LayoutArgs& a, const diffkv_layout* L)
{
    a.p_max = L->p_max;
    a.page_bytes = L->page_bytes;
    a.tsh = 0;
    for (int p = 0; p < 2; ++p) {
        a.T[p] = L->tokens_per_page[p];
        a.kb[p] = L->k_bits[p];
        a.vb[p] = L->v_bits[p];
        int sh = 0;
        while ((1 << sh) < a.T[p]) ++sh;
        a.tsh |= sh << (8 * p);
        a.off_kcode[p] = L->off_kcode[p];
        a.off_kmeta[p] = L->off_kmeta[p];
        a.off_vcode[p] = L->off_vcode[p];
        a.off_vmeta[p] = L->off_vmeta[p];
        a.off_score[p] = L->off_score[p];
        a.off_pos[p] = L->off_pos[p];
    }
}

struct AppendWs {
    int64_t flags, tstate, sold, row_off, ord, tplan, job_table, total;
    int64_t max_jobs;  // bound on the call's page jobs (sizes the commit grid and the job map)
};

AppendWs append_ws(int64_t B, int64_t Hkv, int64_t total_new)
{
    AppendWs w;
    const int64_t T = B * Hkv;
    w.max_jobs = Hkv * ((3 * total_new + 31) / 32 + 4 * B);
    const bool planned = append_planned(B, Hkv);
    int64_t o = 0;
    w.flags = o;   o = align256(o + (int64_t)sizeof(CallFlags));
    w.tstate = o;  o = align256(o + T * (int64_t)sizeof(TState));
    w.sold = o;    o = align256(o + B * 4);
    w.row_off = o; o = align256(o + B * 4);
    w.ord = o;     o = align256(o + total_new * Hkv * 4);
    w.tplan = o;   o = align256(o + (planned ? T * 8 : 0));
    w.job_table = o; o = align256(o + (planned ? w.max_jobs * 4 : 0));
    w.total = o;
    return w;
}

// Attention workspace: one arrival word per table (split tables count their
// shares' partial states in it), then the partial states: automatic (0) or
// balanced (-1) mode one per (share, table) slot k + t; split mode (S > 1) S
// per table; S = 1 needs none.
struct AttnWs {
    int64_t arrive, part, total, nparts;
};

AttnWs attn_ws(int64_t B, int64_t Hq, int64_t Hkv, int64_t splits, int64_t workers)
{
    AttnWs w;
    const int64_t T = B * Hkv;
    const int64_t gq = Hkv > 0 ? Hq / Hkv : 1;
    w.nparts = (splits == 0 || splits == -1) ? workers + T : (splits > 1 ? T * splits : 0);
    int64_t o = 0;
    w.arrive = o; o = align256(o + T * 8);
    w.part = o;   o = align256(o + w.nparts * gq * (kD + 2) * 4);
    w.total = o;
    return w;
}

// Prompt significance: sequence offsets and clamped lengths, row log2-sum-exps.
struct PromptWs {
    int64_t off, nlen, lse2, total;
};

PromptWs prompt_ws(int64_t B, int64_t Hq, int64_t total_new)
{
    PromptWs w;
    int64_t o = 0;
    w.off = o;  o = align256(o + B * 8);
    w.nlen = o; o = align256(o + B * 4);
    w.lse2 = o; o = align256(o + total_new * Hq * 4);
    w.total = o;
    return w;
}

int64_t compact_ws(int64_t T) { return align256(sizeof(CallFlags)) + 2 * align256(T * 4); }
int64_t alloc_ws(int64_t T) { return align256(sizeof(CallFlags)) + align256(T * 16); }
// generation step: call flags, per-table actions, page requests and ring offsets
int64_t gen_ws(int64_t T)
{
    return align256(sizeof(CallFlags)) + 2 * align256(T * 16) + 2 * align256(T * 4);
}


// Both attention entry points.  `noalloc`: the workspace is the device's fixed
// scratch, sized for the mode the call resolves to on the current device.
diffkv_status attention_call(const diffkv_layout* layout, const diffkv_cache* cache, int32_t num_q_heads,
                             const uint16_t* q, float sm_scale, float* out, float* lse, int32_t num_splits,
                             void* ws, size_t ws_bytes, bool noalloc, void* stream)
{
    if (!layout_valid(layout) || !cache_valid(cache) || !cache->pool) return DIFFKV_E_INVAL;
    if (num_q_heads <= 0 || num_q_heads % cache->num_kv_heads != 0 || num_splits < -1)
        return DIFFKV_E_INVAL;
    if (!layout_kernels_supported(layout)) return DIFFKV_E_UNSUPPORTED;
    if (num_q_heads / cache->num_kv_heads > 8) return DIFFKV_E_UNSUPPORTED;
    if (cache->num_seqs == 0) return DIFFKV_OK;
    if (!q || !out) return DIFFKV_E_INVAL;
    if (cache->num_seqs > 65535 || cache->num_kv_heads > 65535) return DIFFKV_E_UNSUPPORTED;
    if (num_splits > 65535) return DIFFKV_E_INVAL;
    if ((int64_t)cache->num_seqs * cache->num_kv_heads * (num_splits > 0 ? num_splits : 1) > INT32_MAX)
        return DIFFKV_E_INVAL;
    AttnWs w;
    if (noalloc) {
        const int64_t T = (int64_t)cache->num_seqs * cache->num_kv_heads;
        int mode = 0, workers = 0;
        if (attention_mode(num_q_heads / cache->num_kv_heads, layout_index(layout), T, num_splits, &mode, &workers) !=
            hipSuccess)
            return DIFFKV_E_LAUNCH;
        // the balanced mode writes partial slots share + table < workers + T
        w = attn_ws(cache->num_seqs, num_q_heads, cache->num_kv_heads, mode, workers);
        if (w.total > kNoAllocScratchBytes) return DIFFKV_E_SCRATCH;
        if (noalloc_scratch(&ws) != hipSuccess) return DIFFKV_E_LAUNCH;
        ws_bytes = (size_t)kNoAllocScratchBytes;
    } else {
        w = attn_ws(cache->num_seqs, num_q_heads, cache->num_kv_heads, num_splits, kAttnMaxWorkers);
        if (!ws || (int64_t)ws_bytes < w.total) return DIFFKV_E_WORKSPACE;
    }
    AttnArgs a;
    memset(&a, 0, sizeof(a));
    a.p_max = layout->p_max;
    a.page_bytes = layout->page_bytes;
    a.num_pages = cache->num_pages;
    for (int p = 0; p < 2; ++p) {
        a.off_kcode[p] = layout->off_kcode[p];
        a.off_kmeta[p] = layout->off_kmeta[p];
        a.off_vcode[p] = layout->off_vcode[p];
        a.off_vmeta[p] = layout->off_vmeta[p];
    }
    a.pool = cache->pool;
    a.page_table = cache->page_table;
    a.len = cache->len;
    a.B = cache->num_seqs;
    a.Hkv = cache->num_kv_heads;
    a.Hq = num_q_heads;
    a.q = q;
    a.scale_log2 = sm_scale * 1.4426950408889634f;
    a.out = out;
    a.lse = lse;
    a.splits = num_splits;
    uint8_t* base = static_cast<uint8_t*>(ws);
    a.arrive = reinterpret_cast<unsigned long long*>(base + w.arrive);
    a.part = reinterpret_cast<float*>(base + w.part);
    a.layout = layout_index(layout);
    hipError_t e = launch_attention(a, static_cast<hipStream_t>(stream));
    return e == hipSuccess ? DIFFKV_OK : DIFFKV_E_LAUNCH;
}

}  // namespace

extern "C" {

diffkv_status diffkv_layout_init(diffkv_layout* out, int32_t head_dim, int32_t group,
                                 const int32_t k_bits[2], const int32_t v_bits[2],
                                 const int32_t tokens_per_page[2], int32_t max_seq_len)
{
    return fill_layout(out, head_dim, group, k_bits, v_bits, tokens_per_page, max_seq_len);
}

diffkv_status diffkv_workspace_size(int32_t op, const diffkv_layout* layout, int32_t num_seqs,
                                    int32_t num_q_heads, int32_t num_kv_heads, int64_t total_new,
                                    int32_t num_splits, size_t* bytes)
{
    if (!bytes || !layout_valid(layout) || num_seqs < 0) return DIFFKV_E_INVAL;
    switch (op) {
    case DIFFKV_OP_APPEND:
        if (num_kv_heads <= 0 || total_new < 0) return DIFFKV_E_INVAL;
        *bytes = (size_t)append_ws(num_seqs, num_kv_heads, total_new).total;
        return DIFFKV_OK;
    case DIFFKV_OP_ATTENTION: {
        if (num_q_heads <= 0 || num_kv_heads <= 0 || num_splits < -1) return DIFFKV_E_INVAL;
        *bytes = (size_t)attn_ws(num_seqs, num_q_heads, num_kv_heads, num_splits, kAttnMaxWorkers).total;
        return DIFFKV_OK;
    }
    case DIFFKV_OP_COMPACT:
        if (num_kv_heads <= 0) return DIFFKV_E_INVAL;
        *bytes = (size_t)compact_ws((int64_t)num_seqs * num_kv_heads);
        return DIFFKV_OK;
    case DIFFKV_OP_ALLOC:
        if (num_kv_heads <= 0) return DIFFKV_E_INVAL;
        *bytes = (size_t)alloc_ws((int64_t)num_seqs * num_kv_heads);
        return DIFFKV_OK;
    case DIFFKV_OP_GENERATION:
        if (num_kv_heads <= 0) return DIFFKV_E_INVAL;
        *bytes = (size_t)gen_ws((int64_t)num_seqs * num_kv_heads);
        return DIFFKV_OK;
    case DIFFKV_OP_PROMPT_SIGNIFICANCE:
        if (num_q_heads <= 0 || total_new < 0) return DIFFKV_E_INVAL;
        *bytes = (size_t)prompt_ws(num_seqs, num_q_heads, total_new).total;
        return DIFFKV_OK;
    default:
        return DIFFKV_E_INVAL;
    }
}

diffkv_status diffkv_quantize_append(const diffkv_layout* layout, const diffkv_cache* cache,
                                     int64_t total_new, int32_t max_new, const int32_t* new_len,
                                     const uint16_t* k, const uint16_t* v, const float* score,
                                     const int32_t* quota, float alpha_h, float alpha_l,
                                     int32_t recent_window, void* ws, size_t ws_bytes, void* stream)
{
    if (!layout_valid(layout) || !cache_valid(cache) || !cache->pool || !cache->seq_len)
        return DIFFKV_E_INVAL;
    if (total_new < 0 || max_new < 0 || recent_window < 0) return DIFFKV_E_INVAL;
    if (total_new > INT32_MAX / 4) return DIFFKV_E_INVAL;
    if (!layout_kernels_supported(layout)) return DIFFKV_E_UNSUPPORTED;
    const int64_t B = cache->num_seqs, H = cache->num_kv_heads;
    if (B == 0) return DIFFKV_OK;
    if (!new_len) return DIFFKV_E_INVAL;
    if (total_new > 0 && (!k || !v || !score)) return DIFFKV_E_INVAL;
    if (total_new * H > INT32_MAX) return DIFFKV_E_INVAL;
    const AppendWs w = append_ws(B, H, total_new);
    if (!ws || (int64_t)ws_bytes < w.total) return DIFFKV_E_WORKSPACE;
    if (w.max_jobs > INT32_MAX) return DIFFKV_E_INVAL;
    AppendArgs a;
    memset(&a, 0, sizeof(a));
    fill_layout_args(a, layout);
    a.pool = cache->pool;
    a.num_pages = cache->num_pages;
    a.page_table = cache->page_table;
    a.pages = cache->pages;
    a.len = cache->len;
    a.seq_len = cache->seq_len;
    a.ring = cache->ring;
    a.ring_ptr = cache->ring_ptr;
    a.status = cache->status;
    a.B = (int)B;
    a.Hkv = (int)H;
    a.total_new = total_new;
    a.max_new = max_new;
    a.new_len = new_len;
    a.k = k;
    a.v = v;
    a.score = score;
    a.quota = quota;
    a.alpha_h = alpha_h;
    a.alpha_l = alpha_l;
    a.window = recent_window;
    uint8_t* base = static_cast<uint8_t*>(ws);
    a.flags = reinterpret_cast<CallFlags*>(base + w.flags);
    a.tstate = reinterpret_cast<TState*>(base + w.tstate);
    a.sold = reinterpret_cast<int32_t*>(base + w.sold);
    a.row_off = reinterpret_cast<int32_t*>(base + w.row_off);
    a.ord = reinterpret_cast<int32_t*>(base + w.ord);
    a.tplan = reinterpret_cast<long long*>(base + w.tplan);
    a.job_table = reinterpret_cast<int32_t*>(base + w.job_table);
    a.job_cap = (int)w.max_jobs;
    // without a planning launch every commit workgroup reads all tables' plan
    // state once, so the grid is capped lower; workgroups loop over the jobs
    // beyond it
    const int64_t cap = append_planned(B, H) ? 4096 : 1024;
    int64_t grid = w.max_jobs < cap ? w.max_jobs : cap;
    if (grid < 1) grid = 1;
    hipError_t e = launch_append(a, (int)grid, static_cast<hipStream_t>(stream));
    return e == hipSuccess ? DIFFKV_OK : DIFFKV_E_LAUNCH;
}

diffkv_status diffkv_decode_attention(const diffkv_layout* layout, const diffkv_cache* cache,
                                      int32_t num_q_heads, const uint16_t* q, float sm_scale,
                                      float* out, float* lse, int32_t num_splits, void* ws,
                                      size_t ws_bytes, void* stream)
{
    return attention_call(layout, cache, num_q_heads, q, sm_scale, out, lse, num_splits, ws, ws_bytes,
                           false, stream);
}

diffkv_status diffkv_decode_attention_noalloc(const diffkv_layout* layout, const diffkv_cache* cache,
                                              int32_t num_q_heads, const uint16_t* q, float sm_scale,
                                              float* out, float* lse, int32_t num_splits, void* stream)
{
    return attention_call(layout, cache, num_q_heads, q, sm_scale, out, lse, num_splits, nullptr, 0,
                          true, stream);
}

diffkv_status diffkv_update_significance(const diffkv_layout* layout, const diffkv_cache* cache,
                                        int32_t num_q_heads, const uint16_t* q, float sm_scale,
                                        const float* lse, void* stream)
{
    if (!layout_valid(layout) || !cache_valid(cache) || !cache->pool || !cache->seq_len) return DIFFKV_E_INVAL;
    if (num_q_heads <= 0 || num_q_heads % cache->num_kv_heads != 0) return DIFFKV_E_INVAL;
    if (!layout_kernels_supported(layout)) return DIFFKV_E_UNSUPPORTED;
    if (num_q_heads / cache->num_kv_heads > 8) return DIFFKV_E_UNSUPPORTED;
    if (cache->num_seqs == 0) return DIFFKV_OK;
    if (!q || !lse) return DIFFKV_E_INVAL;
    SigArgs a;
    memset(&a, 0, sizeof(a));
    a.p_max = layout->p_max;
    a.num_pages = cache->num_pages;
    for (int p = 0; p < 2; ++p) {
        a.off_score[p] = layout->off_score[p];
        a.off_pos[p] = layout->off_pos[p];
    }
    a.pool = cache->pool;
    a.page_table = cache->page_table;
    a.len = cache->len;
    a.seq_len = cache->seq_len;
    a.B = cache->num_seqs;
    a.Hkv = cache->num_kv_heads;
    a.Hq = num_q_heads;
    a.q = q;
    a.scale_log2 = sm_scale * 1.4426950408889634f;
    a.lse = lse;
    a.layout = layout_index(layout);
    hipError_t e = launch_significance(a, static_cast<hipStream_t>(stream));
    return e == hipSuccess ? DIFFKV_OK : DIFFKV_E_LAUNCH;
}

diffkv_status diffkv_prompt_significance(const diffkv_layout* layout, int32_t num_seqs, int64_t total_new,
                                        int32_t max_new, const int32_t* new_len, int32_t num_q_heads,
                                        int32_t num_kv_heads, const uint16_t* q, const uint16_t* k,
                                        float sm_scale, const float* lse, float* score, void* ws,
                                        size_t ws_bytes, void* stream)
{
    if (!layout_valid(layout) || num_seqs < 0 || total_new < 0 || max_new < 0) return DIFFKV_E_INVAL;
    if (num_q_heads <= 0 || num_kv_heads <= 0 || num_q_heads % num_kv_heads != 0) return DIFFKV_E_INVAL;
    if (num_q_heads / num_kv_heads > 8) return DIFFKV_E_UNSUPPORTED;
    if (!(sm_scale > 0.0f) || sm_scale > 1e30f) return DIFFKV_E_INVAL;
    if (num_seqs == 0 || total_new == 0 || max_new == 0) return DIFFKV_OK;
    if (!new_len || !q || !k || !score) return DIFFKV_E_INVAL;
    if (((uintptr_t)q | (uintptr_t)k) % 16 != 0) return DIFFKV_E_INVAL;
    const PromptWs w = prompt_ws(num_seqs, num_q_heads, total_new);
    if (!ws || (int64_t)ws_bytes < w.total) return DIFFKV_E_WORKSPACE;
    PromptArgs a;
    memset(&a, 0, sizeof(a));
    a.B = num_seqs;
    a.Hq = num_q_heads;
    a.Hkv = num_kv_heads;
    a.max_new = max_new;
    a.total_new = total_new;
    a.new_len = new_len;
    a.q = q;
    a.k = k;
    a.lse = lse;
    a.scale_log2 = sm_scale * 1.4426950408889634f;
    a.score = score;
    uint8_t* base = static_cast<uint8_t*>(ws);
    a.off = reinterpret_cast<long long*>(base + w.off);
    a.nlen = reinterpret_cast<int32_t*>(base + w.nlen);
    a.lse2 = reinterpret_cast<float*>(base + w.lse2);
    hipError_t e = launch_prompt_significance(a, num_q_heads / num_kv_heads, static_cast<hipStream_t>(stream));
    return e == hipSuccess ? DIFFKV_OK : DIFFKV_E_LAUNCH;
}

diffkv_status diffkv_compact_free_list(const diffkv_layout* layout, const diffkv_cache* cache,
                                       int32_t num_tables, const uint8_t* release, void* ws,
                                       size_t ws_bytes, void* stream)
{
    if (!layout_valid(layout) || !cache_valid(cache)) return DIFFKV_E_INVAL;
    if (num_tables < 0 || (int64_t)num_tables > (int64_t)cache->num_seqs * cache->num_kv_heads)
        return DIFFKV_E_INVAL;
    if (num_tables == 0) return DIFFKV_OK;
    if (!release) return DIFFKV_E_INVAL;
    if (layout->p_max > 8192) return DIFFKV_E_UNSUPPORTED;  // LDS staging of one row
    if ((int64_t)num_tables > (int64_t)1024 * 1024) return DIFFKV_E_UNSUPPORTED;  // count groups
    const int64_t need = compact_ws(num_tables);
    if (!ws || (int64_t)ws_bytes < need) return DIFFKV_E_WORKSPACE;
    CompactArgs a;
    memset(&a, 0, sizeof(a));
    a.p_max = layout->p_max;
    a.T[0] = layout->tokens_per_page[0];
    a.T[1] = layout->tokens_per_page[1];
    a.num_pages = cache->num_pages;
    a.page_table = cache->page_table;
    a.pages = cache->pages;
    a.len = cache->len;
    a.ring = cache->ring;
    a.ring_ptr = cache->ring_ptr;
    a.num_tables = num_tables;
    a.release = release;
    uint8_t* base = static_cast<uint8_t*>(ws);
    a.flags = reinterpret_cast<CallFlags*>(base);
    a.count = reinterpret_cast<int32_t*>(base + align256(sizeof(CallFlags)));
    a.offset = reinterpret_cast<int32_t*>(base + align256(sizeof(CallFlags)) + align256((int64_t)num_tables * 4));
    hipError_t e = launch_compact(a, static_cast<hipStream_t>(stream));
    return e == hipSuccess ? DIFFKV_OK : DIFFKV_E_LAUNCH;
}

diffkv_status diffkv_alloc_pages(const diffkv_layout* layout, const diffkv_cache* cache,
                                 int32_t num_tables, const int32_t* demand, void* ws,
                                 size_t ws_bytes, void* stream)
{
    if (!layout_valid(layout) || !cache_valid(cache)) return DIFFKV_E_INVAL;
    if (num_tables < 0 || (int64_t)num_tables > (int64_t)cache->num_seqs * cache->num_kv_heads)
        return DIFFKV_E_INVAL;
    if (num_tables == 0) return DIFFKV_OK;
    if (!demand) return DIFFKV_E_INVAL;
    const int64_t need = alloc_ws(num_tables);
    if (!ws || (int64_t)ws_bytes < need) return DIFFKV_E_WORKSPACE;
    AllocArgs a;
    memset(&a, 0, sizeof(a));
    a.p_max = layout->p_max;
    a.num_pages = cache->num_pages;
    a.page_table = cache->page_table;
    a.pages = cache->pages;
    a.ring = cache->ring;
    a.ring_ptr = cache->ring_ptr;
    a.status = cache->status;
    a.num_tables = num_tables;
    a.demand = demand;
    uint8_t* base = static_cast<uint8_t*>(ws);
    a.flags = reinterpret_cast<CallFlags*>(base);
    a.tstate = reinterpret_cast<int4*>(base + align256(sizeof(CallFlags)));
    hipError_t e = launch_alloc(a, static_cast<hipStream_t>(stream));
    return e == hipSuccess ? DIFFKV_OK : DIFFKV_E_LAUNCH;
}

diffkv_status diffkv_generation_step(const diffkv_layout* layout, const diffkv_cache* cache,
                                     float alpha_h, float alpha_l, int32_t recent_window, void* ws,
                                     size_t ws_bytes, void* stream)
{
    if (!layout_valid(layout) || !cache_valid(cache) || !cache->pool || !cache->seq_len)
        return DIFFKV_E_INVAL;
    if (recent_window < 0) return DIFFKV_E_INVAL;
    if (layout_index(layout) != 0) return DIFFKV_E_UNSUPPORTED;  // K8V4 / K4V2, 16 / 32 tokens
    const int64_t T = (int64_t)cache->num_seqs * cache->num_kv_heads;
    if (T == 0) return DIFFKV_OK;
    if (!ws || (int64_t)ws_bytes < gen_ws(T)) return DIFFKV_E_WORKSPACE;
    uint8_t* base = static_cast<uint8_t*>(ws);
    GenArgs g;
    memset(&g, 0, sizeof(g));
    fill_layout_args(g, layout);
    g.pool = cache->pool;
    g.num_pages = cache->num_pages;
    g.page_table = cache->page_table;
    g.pages = cache->pages;
    g.len = cache->len;
    g.seq_len = cache->seq_len;
    g.ring = cache->ring;
    g.ring_ptr = cache->ring_ptr;
    g.status = cache->status;
    g.Hkv = cache->num_kv_heads;
    g.num_tables = (int)T;
    g.alpha_h = alpha_h;
    g.alpha_l = alpha_l;
    g.window = recent_window;
    int64_t o = 0;
    g.flags = reinterpret_cast<CallFlags*>(base + o);  o += align256(sizeof(CallFlags));
    g.act = reinterpret_cast<int4*>(base + o);         o += align256(T * 16);
    g.ids = reinterpret_cast<int4*>(base + o);         o += align256(T * 16);
    g.demand = reinterpret_cast<int32_t*>(base + o);   o += align256(T * 4);
    g.offset = reinterpret_cast<int32_t*>(base + o);
    hipError_t e = launch_generation(g, static_cast<hipStream_t>(stream));
    return e == hipSuccess ? DIFFKV_OK : DIFFKV_E_LAUNCH;
}

const char* diffkv_status_str(diffkv_status s)
{
    switch (s) {
    case DIFFKV_OK: return "ok";
    case DIFFKV_E_INVAL: return "invalid argument";
    case DIFFKV_E_UNSUPPORTED: return "layout or shape not supported by the gfx950 kernels";
    case DIFFKV_E_WORKSPACE: return "workspace too small";
    case DIFFKV_E_LAUNCH: return "HIP launch failed";
    case DIFFKV_E_SCRATCH: return "call needs more than the fixed scratch of the no-allocation entry point";
    default: return "unknown status";
    }
}

}  // extern "C"
