// k_memory.hip -- KV compressor, page allocation and free-list compaction
// kernels for gfx950 (DiffKV Sec. 4, Sec. 5.2, Sec. 5.3).
//
// The compressor runs as two launches on the caller's stream:
//   append_classify  one workgroup per table: classes its new tokens (quota
//                    form by a two-target radix select on the score bits, or
//                    the Algorithm 1 threshold comparisons), ranks the kept
//                    tokens of each section in position order;
//   append_commit    every workgroup derives the plan from the classify
//                    results (page demand per table, one prefix sum over
//                    tables, all-or-nothing check against the free region and
//                    the table width); workgroup 0 writes the new state, and
//                    all take (table, section, page) jobs: resolve the page ID
//                    (new pages from the table's ring region), quantize each
//                    token's 32-dim groups and write the page.
// Allocation alone (alloc_plan + alloc_write) and compaction (compact_count,
// compact_scan, compact_apply) follow the same planning/coordination split:
// per-table work is fully parallel, one prefix sum gives every table a
// disjoint ring region.
#include "internal.hpp"

namespace dkv {

// ---------------------------------------------------------------------------
// shared small pieces
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint32_t score_key(float s)
{
    uint32_t u = __float_as_uint(s);
    if (u == 0x80000000u) u = 0;  // -0 == +0
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ __forceinline__ int ceil_div(int a, int b) { return (a + b - 1) / b; }

// ---------------------------------------------------------------------------
// append_classify: grid (Hkv, B), block 1024
// ---------------------------------------------------------------------------
constexpr int kClsThreads = 1024;
constexpr int kClsLdsKeys = 8192;  // tables with more new tokens re-read keys from global

__global__ __launch_bounds__(kClsThreads) void append_classify(AppendArgs a)
{
    const int h = blockIdx.x, b = blockIdx.y;
    const int H = a.Hkv;
    const int t = b * H + h;
    const int tid = threadIdx.x;
    __shared__ long long s_scan[kClsThreads / kWave + 1];
    __shared__ int s_hist[2][256];
    __shared__ int s_sel[4];
    __shared__ uint32_t s_keys[kClsLdsKeys];

    if (t == 0 && tid == 0) {  // ring pointers before this call (the commit kernel moves head)
        a.flags->head_old = a.ring_ptr[0];
        a.flags->tail_old = a.ring_ptr[1];
    }
    // row offset of this sequence (sum of new_len over lower sequences)
    long long part = 0;
    for (int i = tid; i < b; i += kClsThreads) part += a.new_len[i];
    uint32_t unused;
    const long long off_b = block_sum_or(part, 0u, s_scan, &unused);
    const int n = a.new_len[b];
    TState* ts = a.tstate + t;
    const bool bad = n < 0 || n > a.max_new || off_b + n > a.total_new ||
                     (b == a.B - 1 && off_b + n != a.total_new);
    if (tid == 0) {  // section lengths and pages before this call
        ts->lold[0] = a.len[2 * t];
        ts->lold[1] = a.len[2 * t + 1];
        ts->pold[0] = a.pages[2 * t];
        ts->pold[1] = a.pages[2 * t + 1];
    }
    if (bad) {
        if (tid == 0) {  // the commit kernel turns n < 0 into DIFFKV_ST_BAD_INPUT
            ts->cnt[0] = ts->cnt[1] = 0;
            ts->n = -1;
        }
        return;
    }
    if (h == 0 && tid == 0) {
        a.sold[b] = a.seq_len[b];
        a.row_off[b] = (int)off_b;
    }
    const int W = a.window < n ? a.window : n;
    const int avail = n - W;
    const float* sc = a.score + off_b * H + h;
    int32_t* ord = a.ord + off_b * H + (long long)h * n;
    const bool in_lds = avail <= kClsLdsKeys;

    // ---- quota form: two-target radix select (k-th largest key) ----------
    int k_sel[2] = {0, 0};
    uint32_t K[2] = {0, 0};
    int need[2] = {0, 0};
    const bool quota = a.quota != nullptr;
    float thr_h = 0.f, thr_l = 0.f;
    if (quota) {
        const int q0 = a.quota[2 * t], q1 = a.quota[2 * t + 1];
        const int nh = q0 < 0 ? 0 : (q0 > avail ? avail : q0);
        const int nl = q1 < 0 ? 0 : (q1 > avail - nh ? avail - nh : q1);
        k_sel[0] = nh;
        k_sel[1] = nh + nl;
        // a cut that keeps every non-window token needs no selection
        const bool sel0 = nh > 0 && nh < avail, sel1 = nh + nl > 0 && nh + nl < avail;
        if (sel0 || sel1) {
            if (in_lds) {
                for (int j = tid; j < avail; j += kClsThreads) s_keys[j] = score_key(sc[(long long)j * H]);
                __syncthreads();
            }
            uint32_t prefix[2] = {0, 0}, mask = 0;
            int kk[2] = {sel0 ? nh : 0, sel1 ? nh + nl : 0};
            for (int shift = 24; shift >= 0; shift -= 8) {
                for (int i = tid; i < 512; i += kClsThreads) (&s_hist[0][0])[i] = 0;
                __syncthreads();
                for (int j = tid; j < avail; j += kClsThreads) {
                    const uint32_t key = in_lds ? s_keys[j] : score_key(sc[(long long)j * H]);
                    const uint32_t dig = (key >> shift) & 255u;
#pragma unroll
                    for (int s2 = 0; s2 < 2; ++s2)
                        if (kk[s2] > 0 && (key & mask) == prefix[s2]) atomicAdd(&s_hist[s2][dig], 1);
                }
                __syncthreads();
                if (tid < 2 * kWave) {  // two waves find the cut bins with a scan from the top
                    const int s2 = tid / kWave, l = tid & (kWave - 1);
                    if (kk[s2] > 0) {
                        // lane l owns bins 255-4l .. 252-4l (descending)
                        int c[4], tot4 = 0;
#pragma unroll
                        for (int e = 0; e < 4; ++e) { c[e] = s_hist[s2][255 - 4 * l - e]; tot4 += c[e]; }
                        const int incl = wave_incl_scan(tot4);
                        int above = incl - tot4;
                        if (above < kk[s2] && incl >= kk[s2]) {
#pragma unroll
                            for (int e = 0; e < 4; ++e) {
                                if (above + c[e] >= kk[s2]) {
                                    s_sel[2 * s2] = 255 - 4 * l - e;
                                    s_sel[2 * s2 + 1] = above;
                                    break;
                                }
                                above += c[e];
                            }
                        }
                    }
                }
                __syncthreads();
#pragma unroll
                for (int s2 = 0; s2 < 2; ++s2) {
                    if (kk[s2] > 0) {
                        prefix[s2] |= (uint32_t)s_sel[2 * s2] << shift;
                        kk[s2] -= s_sel[2 * s2 + 1];
                    }
                }
                mask |= 255u << shift;
                __syncthreads();
            }
            K[0] = prefix[0];
            K[1] = prefix[1];
            need[0] = kk[0];  // tokens with key == K that still belong above the cut
            need[1] = kk[1];
        }
        // cuts at 0 or at avail: every token is above (or below) them
        if (!sel0) { K[0] = 0; need[0] = nh > 0 ? avail : 0; }
        if (!sel1) { K[1] = 0; need[1] = nh + nl > 0 ? avail : 0; }
        if (!sel0 && nh > 0) k_sel[0] = -1;  // marker: all non-window tokens are high
        if (!sel1 && nh + nl > 0) k_sel[1] = -1;
    } else {
        const float N = (float)(a.seq_len[b] + n);
        thr_h = a.alpha_h / N;
        thr_l = a.alpha_l / N;
    }

    // ---- classes and in-section ranks, in position order ------------------
    long long carry_tie = 0, carry_rank = 0;
    const bool need_ties = quota && (k_sel[0] > 0 || k_sel[1] > 0);
    for (int base = 0; base < n; base += kClsThreads) {
        const int j = base + tid;
        const bool valid = j < n;
        const bool win = valid && j >= avail;
        float s = 0.f;
        uint32_t key = 0;
        if (valid && !win) {
            if (quota && in_lds && need_ties) key = s_keys[j];
            else {
                s = sc[(long long)j * H];
                key = score_key(s);
            }
        }
        bool hi = win, lo = false;
        if (quota) {
            const bool e0 = valid && !win && k_sel[0] > 0 && key == K[0];
            const bool e1 = valid && !win && k_sel[1] > 0 && key == K[1];
            int r0 = 0, r1 = 0;
            if (need_ties) {
                long long tot;
                long long ex = block_excl_scan<long long>((long long)e0 | ((long long)e1 << 32), s_scan, &tot);
                ex += carry_tie;
                carry_tie += tot;
                r0 = (int)(ex & 0xffffffffll);
                r1 = (int)(ex >> 32);
            }
            if (valid && !win) {
                hi = k_sel[0] < 0 || (k_sel[0] > 0 && (key > K[0] || (e0 && r0 < need[0])));
                lo = !hi && (k_sel[1] < 0 || (k_sel[1] > 0 && (key > K[1] || (e1 && r1 < need[1]))));
            }
        } else if (valid && !win) {
            hi = s >= thr_h;
            lo = !hi && s >= thr_l;
        }
        long long tot;
        long long ex = block_excl_scan<long long>((long long)hi | ((long long)lo << 32), s_scan, &tot);
        ex += carry_rank;
        carry_rank += tot;
        if (hi) ord[(int)(ex & 0xffffffffll)] = j;
        if (lo) ord[n - 1 - (int)(ex >> 32)] = j;
    }
    if (tid == 0) {
        ts->cnt[0] = (int)(carry_rank & 0xffffffffll);
        ts->cnt[1] = (int)(carry_rank >> 32);
        ts->n = n;
    }
}

constexpr int kPlanThreads = 1024;

// ---------------------------------------------------------------------------
// append_commit: plan + quantize in one launch.
// Every workgroup first derives the call's plan from the per-table state the
// classify kernel left (new tokens per section, section lengths and pages
// before the call): page demand, page jobs, one prefix sum over tables (ring
// region and first job of every table), and the all-or-nothing checks.  So no
// workgroup waits on another: workgroup 0 writes the new state (lengths,
// pages, seq_len, ring head) while all of them -- reading only the snapshot
// -- take page jobs (table, section, page) in job order.
// ---------------------------------------------------------------------------
// Quantize one 32-dim group spread over 16 lanes (2 values per lane).
// Arithmetic is IEEE fp32 with no contraction, identical to the text of the
// quantizer: s = fp16((max-min)/L), z = fp16(min), code = clamp(rint((x-z)/s)).
__device__ __forceinline__ void quant_pair(uint32_t xbits, int lb, uint32_t& sz, uint32_t& c0,
                                           uint32_t& c1)
{
#pragma clang fp contract(off)
    float x0 = h2f(xbits & 0xffffu) + 0.0f;
    float x1 = h2f(xbits >> 16) + 0.0f;
    float mn = wave_min_w<16>(fminf(x0, x1));
    float mx = wave_max_w<16>(fmaxf(x0, x1));
    float s32 = (mx - mn) / (float)lb;
    uint32_t s16 = f2h_rne(s32);
    uint32_t z16 = f2h_rne(mn);
    float s = h2f(s16), z = h2f(z16);
    if (s16 == 0) {
        c0 = c1 = 0;
    } else {
        float r0 = rintf((x0 - z) / s);
        float r1 = rintf((x1 - z) / s);
        r0 = fminf(fmaxf(r0, 0.0f), (float)lb);
        r1 = fminf(fmaxf(r1, 0.0f), (float)lb);
        c0 = (uint32_t)r0;
        c1 = (uint32_t)r1;
    }
    sz = s16 | (z16 << 16);
}

constexpr int kQuantWaves = 4;
constexpr int kCommitThreads = kQuantWaves * kWave;
constexpr int kTokIlp = 4;    // tokens a wave quantizes side by side
constexpr int kTokLoad = 8;   // tokens a wave loads up front: a 32-token page in one round of loads
static_assert(kTokLoad * kQuantWaves >= 32, "one round of loads per page");

struct TablePlan {
    int need[2], jobs[2];
    bool held_over;  // more pages than p_max after the call
};

__device__ __forceinline__ TablePlan table_plan(const TState& s, const int (&T)[2], int P)
{
    TablePlan tp;
    int held = 0;
#pragma unroll
    for (int sec = 0; sec < 2; ++sec) {
        const int want = ceil_div(s.lold[sec] + s.cnt[sec], T[sec]);
        tp.need[sec] = want > s.pold[sec] ? want - s.pold[sec] : 0;
        held += want > s.pold[sec] ? want : s.pold[sec];
        tp.jobs[sec] = s.cnt[sec] ? (s.lold[sec] + s.cnt[sec] - 1) / T[sec] - s.lold[sec] / T[sec] + 1 : 0;
    }
    tp.held_over = held > P;
    return tp;
}

struct JobDesc {
    int t, sec, p, u0, u1, lold, n, tslot;
    long long ring_idx;  // ring position of a new page, -1 for a page already held
    int id;
};

__global__ __launch_bounds__(kCommitThreads) void append_commit(AppendArgs a)
{
    const int tid = threadIdx.x;
    const int NT = a.B * a.Hkv;
    const int P = a.p_max;
    const int T[2] = {a.T[0], a.T[1]};
    __shared__ long long s_scan[kCommitThreads / kWave + 1];
    __shared__ JobDesc s_job;
    __shared__ uint64_t s_rows[kQuantWaves][kWave][2];
    const long long head_old = a.flags->head_old, tail_old = a.flags->tail_old;

    // ---- the plan, in every workgroup (each thread a contiguous run of tables)
    const int per = (NT + kCommitThreads - 1) / kCommitThreads;
    const int t0 = tid * per;
    const int t1 = t0 + per < NT ? t0 + per : NT;
    long long packed = 0;  // new pages | jobs << 32
    uint32_t bits = 0;
    for (int t = t0; t < t1; ++t) {
        const TState s = a.tstate[t];
        if (s.n < 0) {
            bits |= DIFFKV_ST_BAD_INPUT;
            continue;
        }
        const TablePlan tp = table_plan(s, T, P);
        if (tp.held_over) bits |= DIFFKV_ST_TABLE_OVERFLOW;
        packed += (tp.need[0] + tp.need[1]) | ((long long)(tp.jobs[0] + tp.jobs[1]) << 32);
    }
    long long tot;
    const long long before = block_excl_scan<long long>(packed, s_scan, &tot);
    // __syncthreads_or returns whether any thread's value is nonzero: one call per bit
    const bool any_bad = __syncthreads_or((int)(bits & DIFFKV_ST_BAD_INPUT));
    const bool any_ovf = __syncthreads_or((int)(bits & DIFFKV_ST_TABLE_OVERFLOW));
    bits = (any_bad ? DIFFKV_ST_BAD_INPUT : 0u) | (any_ovf ? DIFFKV_ST_TABLE_OVERFLOW : 0u);
    const long long total_need = tot & 0xffffffffll;
    const int njobs = (int)(tot >> 32);
    if (bits & DIFFKV_ST_BAD_INPUT) bits = DIFFKV_ST_BAD_INPUT;
    else if (total_need > tail_old - head_old) bits |= DIFFKV_ST_OUT_OF_PAGES;
    if (bits) {  // all or nothing: no state, table or page changes
        if (blockIdx.x == 0 && tid == 0) atomicOr(a.status, bits);
        return;
    }

    // ---- workgroup 0: the state after the call -------------------------------
    if (blockIdx.x == 0) {
        for (int t = t0; t < t1; ++t) {
            const TState s = a.tstate[t];
            const TablePlan tp = table_plan(s, T, P);
#pragma unroll
            for (int sec = 0; sec < 2; ++sec) {
                a.len[2 * t + sec] = s.lold[sec] + s.cnt[sec];
                a.pages[2 * t + sec] = s.pold[sec] + tp.need[sec];
            }
        }
        for (int b = tid; b < a.B; b += kCommitThreads) a.seq_len[b] = a.sold[b] + a.new_len[b];
        if (tid == 0) a.ring_ptr[0] = head_old + total_need;
    }

    // ---- page jobs ------------------------------------------------------------
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = threadIdx.x / kWave;
    const int grp = lane >> 4;
    const int H = a.Hkv;
    const long long page_bytes = a.page_bytes;
    for (int job = blockIdx.x; job < njobs; job += gridDim.x) {
        // the thread whose run of tables holds this job describes it
        long long pre = before;
        for (int t = t0; t < t1; ++t) {
            const TState s = a.tstate[t];
            const TablePlan tp = table_plan(s, T, P);
            const int jo = (int)(pre >> 32);
            if (jo <= job && job < jo + tp.jobs[0] + tp.jobs[1]) {
                const int lj = job - jo;
                const int sec = lj < tp.jobs[0] ? 0 : 1;
                const int p = s.lold[sec] / T[sec] + (sec ? lj - tp.jobs[0] : lj);
                const int lo = s.lold[sec], hi_end = s.lold[sec] + s.cnt[sec];
                s_job.t = t;
                s_job.sec = sec;
                s_job.p = p;
                s_job.u0 = lo > p * T[sec] ? lo : p * T[sec];
                s_job.u1 = hi_end < (p + 1) * T[sec] ? hi_end : (p + 1) * T[sec];
                s_job.lold = lo;
                s_job.n = s.n;
                s_job.tslot = sec ? P - 1 - p : p;
                // a new page comes from this table's ring region, high pages first
                s_job.ring_idx = p < s.pold[sec] ? -1
                                                 : head_old + (pre & 0xffffffffll) + (sec ? tp.need[0] : 0) + (p - s.pold[sec]);
            }
            pre += (tp.need[0] + tp.need[1]) | ((long long)(tp.jobs[0] + tp.jobs[1]) << 32);
        }
        __syncthreads();
        const int t = s_job.t, sec = s_job.sec, p = s_job.p, u0 = s_job.u0, u1 = s_job.u1;
        const int lold = s_job.lold, n = s_job.n;
        const int b = t / H, h = t - b * H;
        const int TT = T[sec];
        const int kb = sec ? 4 : 8, vb = sec ? 2 : 4;
        // one thread resolves the page ID while the others load their tokens
        if (tid == 0) {
            int32_t* trow = a.page_table + (long long)t * P;
            int id;
            if (s_job.ring_idx < 0) {
                id = trow[s_job.tslot];
            } else {
                id = a.ring[s_job.ring_idx % a.num_pages];
                trow[s_job.tslot] = id;
            }
            s_job.id = id;
        }
        // this wave's tokens u0 + wave + kQuantWaves*i, all loaded up front; token
        // u of the section is row ord[u - lold] (high, rank order) or
        // ord[n - 1 - (u - lold)] (low ranks are stored from the back)
        const int off_b = a.row_off[b];
        const int32_t* ord = a.ord + (long long)off_b * H + (long long)h * n;
        int jj[kTokLoad];
        uint32_t kx[kTokLoad], vx[kTokLoad];
#pragma unroll
        for (int i = 0; i < kTokLoad; ++i) {
            const int u = u0 + wave + i * kQuantWaves;
            const int r = (u < u1 ? u : u0) - lold;
            jj[i] = sec ? ord[n - 1 - r] : ord[r];
        }
#pragma unroll
        for (int i = 0; i < kTokLoad; ++i) {
            const long long row = (long long)(off_b + jj[i]) * H + h;
            kx[i] = reinterpret_cast<const uint32_t*>(a.k + row * kD)[lane];
            vx[i] = reinterpret_cast<const uint32_t*>(a.v + row * kD)[lane];
        }
        const int off_kc = a.off_kcode[sec], off_km = a.off_kmeta[sec];
        const int off_vc = a.off_vcode[sec], off_vm = a.off_vmeta[sec];
        const bool fresh = (u0 == p * TT);
        uint8_t* pg = nullptr;
        bool page_ok = false;
        uint64_t row0 = 0, row1 = 0;
        // two passes of kTokIlp tokens: quantize side by side, then store
#pragma unroll
        for (int pass = 0; pass < kTokLoad / kTokIlp; ++pass) {
            const int base_u = u0 + wave + pass * kTokIlp * kQuantWaves;
            if (u0 + pass * kTokIlp * kQuantWaves >= u1) break;  // uniform: no token of this pass in the page
            uint32_t ksz[kTokIlp], kc0[kTokIlp], kc1[kTokIlp], vsz[kTokIlp], vc0[kTokIlp], vc1[kTokIlp];
#pragma unroll
            for (int i = 0; i < kTokIlp; ++i) {
                quant_pair(kx[pass * kTokIlp + i], (1 << kb) - 1, ksz[i], kc0[i], kc1[i]);
                quant_pair(vx[pass * kTokIlp + i], (1 << vb) - 1, vsz[i], vc0[i], vc1[i]);
            }
            if (pass == 0) {
                __syncthreads();  // the page ID is in LDS
                const int id = s_job.id;
                page_ok = (unsigned)id < (unsigned)a.num_pages;  // never write outside the pool
                pg = a.pool + (long long)(page_ok ? id : 0) * page_bytes;
                if (page_ok && fresh) {
                    // A fresh page reads as zero wherever no token lies: zero the token
                    // slots from u1 on in every per-token segment and the page tail.
                    // These bytes are disjoint from the ones the tokens write (V code
                    // rows are written whole, zeros included), so the stores need no
                    // ordering among themselves.
                    const int s_end = u1 - p * TT, nfill = TT - s_end;
                    const uint4 z4 = make_uint4(0, 0, 0, 0);
                    for (int i = tid; i < (kb + 1) * nfill; i += kCommitThreads) {
                        const int c = i / nfill, sl = s_end + (i - c * nfill);  // K chunks (kb per token), then K meta
                        uint8_t* dst = c < kb ? pg + off_kc + (c * TT + sl) * 16 : pg + off_km + sl * 16;
                        *reinterpret_cast<uint4*>(dst) = z4;
                    }
                    for (int i = tid; i < (kNG + 2) * nfill; i += kCommitThreads) {
                        const int g = i / nfill, sl = s_end + (i - g * nfill);  // V meta groups, score, pos
                        uint8_t* dst = g < kNG ? pg + off_vm + (g * TT + sl) * 4
                                               : pg + (g == kNG ? a.off_score[sec] : a.off_pos[sec]) + sl * 4;
                        *reinterpret_cast<uint32_t*>(dst) = 0;
                    }
                    for (long long o = a.off_pos[sec] + (long long)TT * 4 + tid * 16; o < page_bytes;
                         o += kCommitThreads * 16)
                        *reinterpret_cast<uint4*>(pg + o) = z4;
                }
            }
#pragma unroll
            for (int i = 0; i < kTokIlp; ++i) {
                const int u = base_u + i * kQuantWaves;
                if (u >= u1) break;
                const int sl = u - p * TT;
                row0 |= (uint64_t)vc0[i] << (sl * vb);
                row1 |= (uint64_t)vc1[i] << (sl * vb);
                if (!page_ok) continue;
                const long long row = (long long)(off_b + jj[pass * kTokIlp + i]) * H + h;
                if (kb == 8) {
                    uint16_t* dst = reinterpret_cast<uint16_t*>(pg + off_kc + ((lane >> 3) * TT + sl) * 16 +
                                                                ((2 * lane) & 15));
                    *dst = (uint16_t)(kc0[i] | (kc1[i] << 8));
                } else {
                    uint8_t* dst = pg + off_kc + (grp * TT + sl) * 16 + (lane & 15);
                    *dst = (uint8_t)(kc0[i] | (kc1[i] << 4));
                }
                if ((lane & 15) == 0) {
                    *reinterpret_cast<uint32_t*>(pg + off_km + (sl * kNG + grp) * 4) = ksz[i];
                    *reinterpret_cast<uint32_t*>(pg + off_vm + (grp * TT + sl) * 4) = vsz[i];
                }
                if (lane == 0) {
                    reinterpret_cast<float*>(pg + a.off_score[sec])[sl] = a.score[row];
                    reinterpret_cast<int32_t*>(pg + a.off_pos[sec])[sl] = a.sold[b] + jj[pass * kTokIlp + i];
                }
            }
        }
        // the page's dimension-major V code rows: OR of the waves' bits (and of the
        // bits already on a page being continued), one store per dimension pair
        s_rows[wave][lane][0] = row0;
        s_rows[wave][lane][1] = row1;
        __syncthreads();
        if (wave == 0 && page_ok) {
            uint64_t r0 = 0, r1 = 0;
            if (!fresh) {
                const uint4 r = *reinterpret_cast<const uint4*>(pg + off_vc + lane * 16);
                r0 = ((uint64_t)r.y << 32) | r.x;
                r1 = ((uint64_t)r.w << 32) | r.z;
            }
#pragma unroll
            for (int w = 0; w < kQuantWaves; ++w) {
                r0 |= s_rows[w][lane][0];
                r1 |= s_rows[w][lane][1];
            }
            *reinterpret_cast<uint4*>(pg + off_vc + lane * 16) =
                make_uint4((uint32_t)r0, (uint32_t)(r0 >> 32), (uint32_t)r1, (uint32_t)(r1 >> 32));
        }
        __syncthreads();  // s_job and s_rows are reused by the next job
    }
}

// ---------------------------------------------------------------------------
// Allocation alone: alloc_plan (one workgroup) + alloc_write (wave per table)
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kPlanThreads) void alloc_plan(AllocArgs a)
{
    const int tid = threadIdx.x;
    const int NT = a.num_tables;
    __shared__ long long s_scan[kPlanThreads / kWave + 1];
    __shared__ long long s_head, s_tail;
    if (tid == 0) {
        s_head = a.ring_ptr[0];
        s_tail = a.ring_ptr[1];
    }
    __syncthreads();
    long long total = 0;
    uint32_t flags = 0;
    for (int t = tid; t < NT; t += kPlanThreads) {
        int d0 = a.demand[2 * t], d1 = a.demand[2 * t + 1];
        if (d0 < 0 || d1 < 0) flags |= DIFFKV_ST_BAD_INPUT;
        total += (long long)(d0 > 0 ? d0 : 0) + (d1 > 0 ? d1 : 0);
        if ((long long)a.pages[2 * t] + a.pages[2 * t + 1] + d0 + d1 > a.p_max)
            flags |= DIFFKV_ST_TABLE_OVERFLOW;
    }
    uint32_t bits;
    const long long total_all = block_sum_or(total, flags, s_scan, &bits);
    if (total_all > s_tail - s_head) bits |= DIFFKV_ST_OUT_OF_PAGES;
    if (bits) {
        if (tid == 0) {
            atomicOr(a.status, bits);
            a.flags->ok = 0;
        }
        return;
    }
    long long carry = 0;
    for (int t0 = 0; t0 < NT; t0 += kPlanThreads) {
        const int t = t0 + tid;
        int d0 = 0, d1 = 0;
        if (t < NT) {
            d0 = a.demand[2 * t];
            d1 = a.demand[2 * t + 1];
        }
        long long tr;
        long long off = block_excl_scan<long long>(d0 + d1, s_scan, &tr) + carry;
        carry += tr;
        if (t < NT) {
            int4 st = make_int4(a.pages[2 * t], a.pages[2 * t + 1], (int)off, d0);
            a.tstate[t] = st;
            a.pages[2 * t] = st.x + d0;
            a.pages[2 * t + 1] = st.y + d1;
        }
    }
    if (tid == 0) {
        a.flags->head_old = s_head;
        a.flags->ok = 1;
        a.ring_ptr[0] = s_head + carry;
    }
}

__global__ __launch_bounds__(kWave) void alloc_write(AllocArgs a)
{
    if (!a.flags->ok) return;
    const int t = blockIdx.x;
    const int4 st = a.tstate[t];
    const int d1 = a.pages[2 * t + 1] - st.y;
    const long long base = a.flags->head_old + st.z;
    int32_t* row = a.page_table + (long long)t * a.p_max;
    for (int i = threadIdx.x; i < st.w; i += kWave) row[st.x + i] = a.ring[(base + i) % a.num_pages];
    for (int i = threadIdx.x; i < d1; i += kWave)
        row[a.p_max - 1 - (st.y + i)] = a.ring[(base + st.w + i) % a.num_pages];
}

// ---------------------------------------------------------------------------
// Compaction: compact_count (wave per table), compact_scan (one workgroup),
// compact_apply (wave per table)
// ---------------------------------------------------------------------------
__device__ __forceinline__ bool slot_live(int slot, int ph, int pl, int P)
{
    return slot < ph || slot >= P - pl;
}

__global__ __launch_bounds__(kWave) void compact_count(CompactArgs a)
{
    const int t = blockIdx.x;
    const int P = a.p_max;
    int ph = a.pages[2 * t], pl = a.pages[2 * t + 1];
    ph = ph < 0 ? 0 : (ph > P ? P : ph);
    pl = pl < 0 ? 0 : (pl > P - ph ? P - ph : pl);
    const uint8_t* rel = a.release + (long long)t * P;
    int c = 0;
    for (int s = threadIdx.x; s < P; s += kWave) c += (rel[s] != 0 && slot_live(s, ph, pl, P));
    c = wave_isum_w<kWave>(c);
    if (threadIdx.x == 0) a.count[t] = c;
}

__global__ __launch_bounds__(kPlanThreads) void compact_scan(CompactArgs a)
{
    const int tid = threadIdx.x;
    __shared__ long long s_scan[kPlanThreads / kWave + 1];
    __shared__ long long s_tail;
    if (tid == 0) s_tail = a.ring_ptr[1];
    __syncthreads();
    long long carry = 0;
    for (int t0 = 0; t0 < a.num_tables; t0 += kPlanThreads) {
        const int t = t0 + tid;
        const int c = t < a.num_tables ? a.count[t] : 0;
        long long tr;
        long long off = block_excl_scan<long long>(c, s_scan, &tr) + carry;
        carry += tr;
        if (t < a.num_tables) a.offset[t] = (int)off;
    }
    if (tid == 0) {
        a.flags->tail_old = s_tail;
        a.ring_ptr[1] = s_tail + carry;
    }
}

// One wave per table; the live part of the row is staged in LDS (dynamic
// shared memory of 2*p_max ints) so the squeeze can write in place.
__global__ __launch_bounds__(kWave) void compact_apply(CompactArgs a)
{
    extern __shared__ int32_t s_row[];  // [0, P): old IDs, [P, 2P): new row
    const int t = blockIdx.x;
    const int lane = threadIdx.x;
    const int P = a.p_max;
    int ph = a.pages[2 * t], pl = a.pages[2 * t + 1];
    ph = ph < 0 ? 0 : (ph > P ? P : ph);  // same clamp as compact_count
    pl = pl < 0 ? 0 : (pl > P - ph ? P - ph : pl);
    const int len0 = a.len[2 * t], len1 = a.len[2 * t + 1];
    const int T0 = a.T[0], T1 = a.T[1];
    const uint8_t* rel = a.release + (long long)t * P;
    int32_t* row = a.page_table + (long long)t * P;
    int32_t* s_new = s_row + P;
    const long long base = a.flags->tail_old + a.offset[t];
    const uint64_t below = (1ull << lane) - 1ull;
    for (int s = lane; s < ph; s += kWave) s_row[s] = row[s];
    for (int s = P - pl + lane; s < P; s += kWave) s_row[s] = row[s];
    __syncthreads();
    // released IDs to the ring in ascending slot order; kept high IDs packed left
    int rank = 0, hi_keep = 0, drop0 = 0, drop1 = 0;
    for (int c = 0; c < ph; c += kWave) {
        const int s = c + lane;
        const bool live = s < ph;
        const bool r = live && rel[s] != 0;
        const uint64_t mr = __ballot(r);
        const uint64_t mk = __ballot(live && !r);
        if (r) {
            a.ring[(base + rank + __popcll(mr & below)) % a.num_pages] = s_row[s];
            int f = len0 - s * T0;
            drop0 += f < 0 ? 0 : (f > T0 ? T0 : f);
        }
        if (live && !r) s_new[hi_keep + __popcll(mk & below)] = s_row[s];
        rank += __popcll(mr);
        hi_keep += __popcll(mk);
    }
    for (int c = P - pl; c < P; c += kWave) {
        const int s = c + lane;
        const bool r = s < P && rel[s] != 0;
        const uint64_t mr = __ballot(r);
        if (r) {
            a.ring[(base + rank + __popcll(mr & below)) % a.num_pages] = s_row[s];
            int f = len1 - (P - 1 - s) * T1;
            drop1 += f < 0 ? 0 : (f > T1 ? T1 : f);
        }
        rank += __popcll(mr);
    }
    // kept low IDs packed right, in section order (section page k sits at slot P-1-k)
    int lo_keep = 0;
    for (int c = 0; c < pl; c += kWave) {
        const int k = c + lane;
        const int s = P - 1 - k;
        const bool keep = k < pl && rel[s] == 0;
        const uint64_t mk = __ballot(keep);
        if (keep) s_new[P - 1 - (lo_keep + __popcll(mk & below))] = s_row[s];
        lo_keep += __popcll(mk);
    }
    __syncthreads();
    for (int s = lane; s < ph; s += kWave) row[s] = s < hi_keep ? s_new[s] : -1;
    for (int s = P - pl + lane; s < P; s += kWave) row[s] = s >= P - lo_keep ? s_new[s] : -1;
    drop0 = wave_isum_w<kWave>(drop0);
    drop1 = wave_isum_w<kWave>(drop1);
    if (lane == 0) {
        a.pages[2 * t] = hi_keep;
        a.pages[2 * t + 1] = lo_keep;
        a.len[2 * t] = len0 - drop0;
        a.len[2 * t + 1] = len1 - drop1;
    }
}

// ---------------------------------------------------------------------------
// launchers
// ---------------------------------------------------------------------------
hipError_t launch_append(const AppendArgs& a, int grid_quant, hipStream_t st)
{
    hipLaunchKernelGGL(append_classify, dim3(a.Hkv, a.B), dim3(kClsThreads), 0, st, a);
    hipLaunchKernelGGL(append_commit, dim3(grid_quant), dim3(kCommitThreads), 0, st, a);
    return hipGetLastError();
}

hipError_t launch_alloc(const AllocArgs& a, hipStream_t st)
{
    hipLaunchKernelGGL(alloc_plan, dim3(1), dim3(kPlanThreads), 0, st, a);
    if (a.num_tables > 0) hipLaunchKernelGGL(alloc_write, dim3(a.num_tables), dim3(kWave), 0, st, a);
    return hipGetLastError();
}

hipError_t launch_compact(const CompactArgs& a, hipStream_t st)
{
    if (a.num_tables == 0) return hipSuccess;
    hipLaunchKernelGGL(compact_count, dim3(a.num_tables), dim3(kWave), 0, st, a);
    hipLaunchKernelGGL(compact_scan, dim3(1), dim3(kPlanThreads), 0, st, a);
    hipLaunchKernelGGL(compact_apply, dim3(a.num_tables), dim3(kWave),
                       (size_t)2 * a.p_max * sizeof(int32_t), st, a);
    return hipGetLastError();
}

}  // namespace dkv
