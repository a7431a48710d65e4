"""Pins of the oracle's classing, page layout, allocation and compaction (CPU only).

Paper anchors: Sec. 1 / Fig. mem_usage_patterns (memory accounting),
Sec. 4 (token classes), Sec. 5.2 (unified pages, circular free page list,
bidirectional page table, table size example), Sec. 5.3 (prompt-phase
worked example).  Where the text fixes no value, invariants and brute force
pin the functions.
"""
import itertools
import json
import os

import numpy as np
import pytest

GOLD = os.path.join(os.path.dirname(__file__), "golden")


# ------------------------------------------------------------ layout ----
def test_layout_sizes(orc):
    L = orc.layout(max_seq_len=4096)
    # high page: 16 tokens K8V4; low page: 32 tokens K4V2 (64-byte aligned segments)
    assert L.used_bytes[0] == 2048 + 256 + 1024 + 256 + 64 + 64 == 3712
    assert L.used_bytes[1] == 2048 + 512 + 1024 + 512 + 128 + 128 == 4352
    assert L.page_bytes == 4352
    assert L.p_max == 257
    # bytes attention reads per token: codes + fp16 scale/zero per 32-dim group
    hi = (L.off_score[0] - L.off_kcode[0]) / 16
    lo = (L.off_score[1] - L.off_kcode[1]) / 32
    assert (hi, lo) == (224.0, 128.0)


def test_table_size_example(orc):
    """Sec. 5.2: batch 128 on Llama3-8B (32 layers x 8 KV heads): all tables take 32 MB.
    The text sizes a table as max_len / tokens-per-high-page entries; with 16 tokens per
    high page that is 256 int32 entries, i.e. max_len 4096.  This build adds one slot
    (a table holding a partial high page and a partial low page needs it), so the
    paper's figure is p_max - 1 entries per table."""
    L = orc.layout(max_seq_len=4096)
    tables = 128 * 32 * 8
    assert tables * (L.p_max - 1) * 4 == 32 * 2 ** 20


def test_p_max_never_overflows(orc):
    """ceil(h/Th) + ceil(l/Tl) <= p_max for every split of max_len tokens (brute force)."""
    for th, tl, mx in [(16, 32, 200), (16, 16, 130), (2, 4, 9), (4, 8, 37)]:
        L = orc.layout(tokens_per_page=(th, tl), max_seq_len=mx)
        worst = max(-(-h // th) + -(-l // tl) for h in range(mx + 1) for l in range(mx + 1 - h))
        assert worst <= L.p_max
        assert worst == L.p_max or mx % th != 0


def test_fig1_memory_accounting(orc):
    g = json.load(open(os.path.join(GOLD, "fig1_memory_usage.json")))
    L = orc.layout()
    fr = []
    for h in g["heads"]:
        n = h["n_high"] + h["n_low"] + h["n_pruned"]
        kf, vf = orc.kv_bits_fraction(L, h["n_high"], h["n_low"], n)
        assert kf == pytest.approx(h["k_frac"], abs=1e-12)
        assert vf == pytest.approx(h["v_frac"], abs=1e-12)
        fr += [kf, vf]
    assert round(np.mean(fr), 3) == g["average_printed"]
    L8 = orc.layout(k_bits=(8, 8), v_bits=(8, 8), tokens_per_page=(16, 16))
    assert orc.kv_bits_fraction(L8, 5, 0, 5) == (g["uniform_int8"], g["uniform_int8"])


# ----------------------------------------------------------- classing ----
def _brute_classes(score, nh, nl, window):
    n = len(score)
    avail = n - min(window, n)
    order = sorted(range(avail), key=lambda j: (-float(score[j]), j))
    nh = min(max(nh, 0), avail)
    nl = min(max(nl, 0), avail - nh)
    cls = np.full(n, 0, np.int8)
    for r, j in enumerate(order):
        cls[j] = 0 if r < nh else (1 if r < nh + nl else -1)
    return cls


def test_classify_quota_brute_force(orc):
    rng = np.random.default_rng(5)
    for trial in range(3000):
        n = int(rng.integers(1, 12))
        # few distinct values -> many ties, incl. signed zeros
        vals = np.array([0.0, -0.0, 0.25, 0.5, 1.0, -1.0], np.float32)
        score = vals[rng.integers(0, len(vals), n)]
        nh, nl = int(rng.integers(-1, n + 3)), int(rng.integers(-1, n + 3))
        w = int(rng.integers(0, 4))
        got = orc.classify(score, quota=(nh, nl), window=w)
        assert np.array_equal(got, _brute_classes(score, nh, nl, w)), (score, nh, nl, w)


def test_classify_quota_invariants(orc):
    rng = np.random.default_rng(6)
    for trial in range(300):
        n = int(rng.integers(1, 400))
        score = rng.random(n).astype(np.float32)
        score[rng.integers(0, n, n // 4)] = score[0]  # ties
        nh, nl = int(rng.integers(0, n)), int(rng.integers(0, n))
        cls = orc.classify(score, quota=(nh, nl))
        nh_c = min(nh, n)
        nl_c = min(nl, n - nh_c)
        assert (cls == 0).sum() == nh_c and (cls == 1).sum() == nl_c
        # monotone in (score, -position): a higher class never ranks below a lower one
        rank = np.array([0, 1, 2])[np.where(cls == -1, 2, cls)]
        for a in range(n):
            better = (score > score[a]) | ((score == score[a]) & (np.arange(n) < a))
            assert np.all(rank[better] <= rank[a])


def test_classify_threshold_boundaries(orc):
    N = 37
    ah, al = 3.0, 0.5
    th, tl = np.float32(ah) / np.float32(N), np.float32(al) / np.float32(N)
    s = np.array([th, np.nextafter(th, 0, dtype=np.float32), tl,
                  np.nextafter(tl, 0, dtype=np.float32), 0.0, 1.0], np.float32)
    cls = orc.classify(s, alpha_h=ah, alpha_l=al, seq_len_after=N)
    assert cls.tolist() == [0, 1, 1, -1, -1, 0]
    # alpha_l = 0 prunes nothing among non-negative scores
    cls = orc.classify(s, alpha_h=ah, alpha_l=0.0, seq_len_after=N)
    assert cls.tolist() == [0, 1, 1, 1, 1, 0]
    # the window's tokens stay high whatever their score
    cls = orc.classify(np.zeros(6, np.float32), alpha_h=ah, alpha_l=al, seq_len_after=N, window=2)
    assert cls.tolist() == [-1, -1, -1, -1, 0, 0]


# ---------------------------------------------- prompt-phase example ----
def test_prompt_phase_worked_example(orc):
    """Sec. 5.3, Fig. memory_management_flow: conservative allocation, planning, recycling."""
    g = json.load(open(os.path.join(GOLD, "prompt_phase_example.json")))
    L = orc.layout(tokens_per_page=tuple(g["tokens_per_page"]), max_seq_len=6)
    assert L.p_max == 4
    c = orc.Cache(L, len(g["ring"]), 1, 2, ring=np.array(g["ring"]))
    c.ring_ptr[:] = g["ring_ptr_before"]
    orc.alloc_pages(c, np.array(g["conservative_demand"]))
    assert c.table.tolist() == g["tables_after_alloc"]
    assert c.ring_ptr.tolist() == g["ring_ptr_after_alloc"]
    # planning: the compressor places each head's tokens into the pages it already holds
    n = g["tokens"]
    rng = np.random.default_rng(0)
    k = (rng.standard_normal((n, 2, 128))).astype(np.float16).view(np.uint16)
    v = (rng.standard_normal((n, 2, 128))).astype(np.float16).view(np.uint16)
    score = rng.permutation(n * 2).reshape(n, 2).astype(np.float32)
    orc.quantize_append(c, np.array([n]), k, v, score, quota=np.array(g["quota"]).reshape(1, 2, 2))
    assert c.ring_ptr.tolist() == g["ring_ptr_after_alloc"]  # no new pages needed
    used = g["used_pages"]
    for t, name in enumerate("AB"):
        hp = -(-c.len[t, 0] // 2)
        lp = -(-c.len[t, 1] // 4)
        assert c.table[t, :hp].tolist() == used[name]["high"]
        assert c.table[t, L.p_max - lp:][::-1].tolist() == used[name]["low"]
    # coordination: recycle the pages the plan left unused
    orc.compact(c, np.array(g["release"], np.uint8))
    assert c.ring[:3].tolist() == g["ring_slots_0_to_2_after"] == g["recycled_in_order"]
    assert c.ring_ptr.tolist() == g["ring_ptr_after_recycle"]
    assert c.table.tolist() == g["tables_after_recycle"]


# ------------------------------------------------------- compaction ----
def _live(c, L):
    out = []
    for t in range(c.num_tables):
        ph, pl = c.pages[t]
        hi = c.table[t, :ph].tolist()
        lo = c.table[t, L.p_max - pl:][::-1].tolist() if pl else []
        out.append((hi, lo))
    return out


def _check_conservation(c, L):
    head, tail = c.ring_ptr
    n = c.num_pages
    assert 0 <= tail - head <= n
    free = [int(c.ring[i % n]) for i in range(head, tail)]
    live = [p for hi, lo in _live(c, L) for p in hi + lo]
    allp = sorted(free + live)
    assert allp == list(range(n)), "every page exactly once in the free region or one table"
    for t in range(c.num_tables):
        ph, pl = c.pages[t]
        mid = c.table[t, ph:L.p_max - pl]
        assert np.all(mid == -1)


def _random_state(orc, rng, tables, num_pages, tokens=(16, 32), p_max_len=200):
    L = orc.layout(tokens_per_page=tokens, max_seq_len=p_max_len)
    c = orc.Cache(L, num_pages, tables, 1, ring=rng.permutation(num_pages), with_pool=False)
    budget = num_pages
    dem = np.zeros((tables, 2), np.int32)
    for t in range(tables):
        a = int(rng.integers(0, min(L.p_max, budget // max(1, tables - t)) + 1))
        hi = int(rng.integers(0, a + 1))
        dem[t] = hi, a - hi
        budget -= a
    orc.alloc_pages(c, dem)
    for t in range(tables):
        for sec, T in enumerate(tokens):
            p = c.pages[t, sec]
            c.len[t, sec] = 0 if p == 0 else (p - 1) * T + int(rng.integers(1, T + 1))
    return L, c


def test_compaction_invariants_random(orc):
    rng = np.random.default_rng(11)
    for trial in range(60):
        L, c = _random_state(orc, rng, int(rng.integers(1, 40)), int(rng.integers(50, 900)))
        for rnd in range(4):
            before = _live(c, L)
            lens = c.len.copy()
            tail0 = int(c.ring_ptr[1])
            head0 = int(c.ring_ptr[0])
            rel = (rng.random((c.num_tables, L.p_max)) < rng.random()).astype(np.uint8)
            orc.compact(c, rel)
            after = _live(c, L)
            released = []
            for t, ((hi, lo), (hi2, lo2)) in enumerate(zip(before, after)):
                ph, pl = len(hi), len(lo)
                rh = [hi[k] for k in range(ph) if rel[t, k]]
                rl_slots = [(L.p_max - 1 - k, lo[k]) for k in range(pl) if rel[t, L.p_max - 1 - k]]
                released += rh + [p for _, p in sorted(rl_slots)]
                assert hi2 == [hi[k] for k in range(ph) if not rel[t, k]]
                assert lo2 == [lo[k] for k in range(pl) if not rel[t, L.p_max - 1 - k]]
                for sec, (sect, T) in enumerate(((hi, 16), (lo, 32))):
                    ks = [k for k in range(len(sect))
                          if rel[t, k if sec == 0 else L.p_max - 1 - k]]
                    fill = sum(min(max(lens[t, sec] - k * T, 0), T) for k in ks)
                    assert c.len[t, sec] == lens[t, sec] - fill
            assert int(c.ring_ptr[1]) - tail0 == len(released)
            assert int(c.ring_ptr[0]) == head0
            ring_new = [int(c.ring[i % c.num_pages]) for i in range(tail0, int(c.ring_ptr[1]))]
            assert ring_new == released
            _check_conservation(c, L)


def test_compaction_brute_force_all_masks(orc):
    """Two tables, up to four live slots each: every release mask."""
    rng = np.random.default_rng(12)
    L = orc.layout(tokens_per_page=(2, 4), max_seq_len=6)
    P = L.p_max
    for dem in [((2, 2), (1, 0)), ((0, 3), (3, 1)), ((1, 1), (2, 2))]:
        for mask_bits in range(1 << (2 * P)):
            c = orc.Cache(L, 13, 2, 1, ring=rng.permutation(13), with_pool=False)
            orc.alloc_pages(c, np.array(dem))
            c.len[:] = c.pages * np.array([2, 4])
            rel = np.array([(mask_bits >> i) & 1 for i in range(2 * P)], np.uint8).reshape(2, P)
            before = _live(c, L)
            orc.compact(c, rel)
            _check_conservation(c, L)
            kept = sum(len(h) + len(l) for h, l in _live(c, L))
            rel_live = sum(int(rel[t, k]) for t in range(2) for k in range(P)
                           if k < dem[t][0] or k >= P - dem[t][1])
            assert kept == sum(map(sum, dem)) - rel_live
            assert before is not None


def test_alloc_all_or_nothing(orc):
    rng = np.random.default_rng(13)
    L, c = _random_state(orc, rng, 8, 100)
    free = int(c.ring_ptr[1] - c.ring_ptr[0])
    snap = c.copy()
    d = np.zeros((8, 2), np.int32)
    d[3, 1] = free + 1
    orc.alloc_pages(c, d)
    assert c.status[0] & 1
    for f in ("table", "pages", "len", "ring", "ring_ptr"):
        assert np.array_equal(getattr(c, f), getattr(snap, f))
    c.status[0] = 0
    d[:] = 0
    d[0, 0] = L.p_max - c.pages[0].sum() + 1
    orc.alloc_pages(c, d)
    assert c.status[0] == 2
    for f in ("table", "pages", "len", "ring", "ring_ptr"):
        assert np.array_equal(getattr(c, f), getattr(snap, f))


# ------------------------------------------- append / page layout -------
def _pack_expected_page(L, sec, slots, orc):
    """Independent packer: builds a page's bytes from per-slot quantizer outputs,
    straight from the layout description (segments, chunk-major keys,
    dimension-major values, little-endian bits)."""
    T = L.tokens_per_page[sec]
    kb, vb = L.k_bits[sec], L.v_bits[sec]
    page = np.zeros(L.page_bytes, np.uint8)
    bits = np.zeros(L.page_bytes * 8, np.uint8)

    def put(byte_off, nbits, val, bitpos=0):
        for i in range(nbits):
            bits[byte_off * 8 + bitpos + i] = (val >> i) & 1

    for slot, (kq, vq, score, pos) in enumerate(slots):
        for d in range(128):
            c = d // (128 // kb)
            e = d % (128 // kb)
            put(L.off_kcode[sec] + (c * T + slot) * 16, kb, int(kq[2][d]), e * kb)
            put(L.off_vcode[sec] + d * (T * vb // 8), vb, int(vq[2][d]), slot * vb)
        for g in range(4):
            put(L.off_kmeta[sec] + (slot * 4 + g) * 4, 16, kq[0][g])
            put(L.off_kmeta[sec] + (slot * 4 + g) * 4 + 2, 16, kq[1][g])
            put(L.off_vmeta[sec] + (g * T + slot) * 4, 16, vq[0][g])
            put(L.off_vmeta[sec] + (g * T + slot) * 4 + 2, 16, vq[1][g])
        put(L.off_score[sec] + slot * 4, 32, int(np.float32(score).view(np.uint32)))
        put(L.off_pos[sec] + slot * 4, 32, int(pos))
    page[:] = np.packbits(bits.reshape(-1, 8), axis=1, bitorder="little").ravel()
    return page


def test_append_page_bytes_match_layout_description(orc):
    rng = np.random.default_rng(21)
    L = orc.layout(max_seq_len=128)
    n = 40
    k = (rng.standard_normal((n, 1, 128)) * 3).astype(np.float16).view(np.uint16)
    v = rng.standard_normal((n, 1, 128)).astype(np.float16).view(np.uint16)
    score = rng.permutation(n).reshape(n, 1).astype(np.float32)
    c = orc.Cache(L, 16, 1, 1)
    c.pool[:] = 0xA5  # garbage in free pages must not leak into a fresh page
    orc.quantize_append(c, np.array([n]), k, v, score, quota=np.array([[[18, 16]]]))
    cls = orc.classify(score[:, 0], quota=(18, 16))
    assert c.len.tolist() == [[18, 16]] and c.pages.tolist() == [[2, 1]]
    for sec in (0, 1):
        toks = [j for j in range(n) if cls[j] == sec]
        T = L.tokens_per_page[sec]
        for p in range(-(-len(toks) // T)):
            slots = []
            for j in toks[p * T:(p + 1) * T]:
                kq = [[], [], np.zeros(128, np.uint8)]
                vq = [[], [], np.zeros(128, np.uint8)]
                for g in range(4):
                    s, z, cd = orc.quantize_group(k[j, 0, 32 * g:32 * g + 32], L.k_bits[sec])
                    kq[0].append(s); kq[1].append(z); kq[2][32 * g:32 * g + 32] = cd
                    s, z, cd = orc.quantize_group(v[j, 0, 32 * g:32 * g + 32], L.v_bits[sec])
                    vq[0].append(s); vq[1].append(z); vq[2][32 * g:32 * g + 32] = cd
                slots.append((kq, vq, score[j, 0], j))
            pid = c.table[0, p] if sec == 0 else c.table[0, L.p_max - 1 - p]
            exp = _pack_expected_page(L, sec, slots, orc)
            assert np.array_equal(c.pool[pid], exp), (sec, p)


def test_append_incremental_equals_bulk(orc):
    """Token-by-token appends (into partial pages) give the same pages as one bulk append."""
    rng = np.random.default_rng(22)
    L = orc.layout(max_seq_len=256)
    n, H = 70, 2
    k = rng.standard_normal((n, H, 128)).astype(np.float16).view(np.uint16)
    v = rng.standard_normal((n, H, 128)).astype(np.float16).view(np.uint16)
    score = rng.random((n, H)).astype(np.float32)
    ring = rng.permutation(64)
    a = orc.Cache(L, 64, 1, H, ring=ring)
    b = orc.Cache(L, 64, 1, H, ring=ring)
    a.pool[:] = 0x5A
    b.pool[:] = 0x5A
    for j in range(n):
        orc.quantize_append(a, np.array([1]), k[j:j + 1], v[j:j + 1], score[j:j + 1],
                            quota=np.full((1, H, 2), [1, 0]))
    orc.quantize_append(b, np.array([n]), k, v, score, quota=np.full((1, H, 2), [n, 0]))
    # the bulk call allocates all of head 0's pages before head 1's; map pages by table slot
    assert np.array_equal(a.len, b.len) and np.array_equal(a.pages, b.pages)
    for t in range(H):
        for p in range(a.pages[t, 0]):
            assert np.array_equal(a.pool[a.table[t, p]], b.pool[b.table[t, p]])


def test_append_threshold_form_over_steps(orc):
    """Generation-phase thresholds shrink with N: token j is high iff score >= alpha_h/(j+1)."""
    rng = np.random.default_rng(25)
    L = orc.layout(max_seq_len=256)
    n, H = 70, 2
    k = rng.standard_normal((n, H, 128)).astype(np.float16).view(np.uint16)
    v = rng.standard_normal((n, H, 128)).astype(np.float16).view(np.uint16)
    score = rng.random((n, H)).astype(np.float32) * 0.05
    a = orc.Cache(L, 64, 1, H, ring=rng.permutation(64))
    for j in range(n):
        orc.quantize_append(a, np.array([1]), k[j:j + 1], v[j:j + 1], score[j:j + 1],
                            alpha_h=1.0, alpha_l=0.5)
    assert a.seq_len[0] == n
    for t in range(H):
        hi = [j for j in range(n) if score[j, t] >= np.float32(1.0) / np.float32(j + 1)]
        lo = [j for j in range(n) if np.float32(0.5) / np.float32(j + 1) <= score[j, t]
              < np.float32(1.0) / np.float32(j + 1)]
        assert [orc.read_token(a, t, 0, u)[3] for u in range(a.len[t, 0])] == hi
        assert [orc.read_token(a, t, 1, u)[3] for u in range(a.len[t, 1])] == lo


def test_append_all_or_nothing(orc):
    rng = np.random.default_rng(23)
    L = orc.layout(max_seq_len=64)
    n, H = 50, 2
    k = rng.standard_normal((n, H, 128)).astype(np.float16).view(np.uint16)
    v = rng.standard_normal((n, H, 128)).astype(np.float16).view(np.uint16)
    score = rng.random((n, H)).astype(np.float32)
    c = orc.Cache(L, 4, 1, H)  # needs 2 high + 1 low page per head -> 6 > 4
    snap = c.copy()
    orc.quantize_append(c, np.array([n]), k, v, score, quota=np.full((1, H, 2), [20, 20]))
    assert c.status[0] == 1
    for f in ("pool", "table", "pages", "len", "seq_len", "ring", "ring_ptr"):
        assert np.array_equal(getattr(c, f), getattr(snap, f)), f
    L2 = orc.layout(max_seq_len=20)  # p_max = 3: 3 high + 1 low pages do not fit
    c = orc.Cache(L2, 64, 1, H)
    snap = c.copy()
    orc.quantize_append(c, np.array([n]), k, v, score, quota=np.full((1, H, 2), [33, 17]))
    assert c.status[0] == 2
    for f in ("pool", "table", "pages", "len", "seq_len", "ring", "ring_ptr"):
        assert np.array_equal(getattr(c, f), getattr(snap, f)), f


def test_append_positions_scores_and_dequant_bound(orc):
    rng = np.random.default_rng(24)
    L = orc.layout(max_seq_len=600)
    B, H = 3, 2
    new_len = np.array([100, 1, 257], np.int32)
    rows = int(new_len.sum())
    k = (rng.standard_normal((rows, H, 128)) * 2).astype(np.float16).view(np.uint16)
    v = rng.standard_normal((rows, H, 128)).astype(np.float16).view(np.uint16)
    score = rng.random((rows, H)).astype(np.float32)
    quota = rng.integers(0, 120, (B, H, 2)).astype(np.int32)
    c = orc.Cache(L, 200, B, H, ring=rng.permutation(200))
    c.seq_len[:] = [5, 0, 9]
    orc.quantize_append(c, new_len, k, v, score, quota=quota, window=3)
    off = np.concatenate([[0], np.cumsum(new_len)])
    for b in range(B):
        for h in range(H):
            t = b * H + h
            n = int(new_len[b])
            cls = orc.classify(score[off[b]:off[b + 1], h], quota=quota[b, h], window=3)
            for sec in (0, 1):
                js = [j for j in range(n) if cls[j] == sec]
                assert c.len[t, sec] == len(js)
                T = L.tokens_per_page[sec]
                assert c.pages[t, sec] == -(-len(js) // T)
                for u, j in enumerate(js):
                    kh, vh, s, pos = orc.read_token(c, t, sec, u)
                    assert pos == [5, 0, 9][b] + j
                    assert s == score[off[b] + j, h]
                    x = k[off[b] + j, h].view(np.float16).astype(np.float64)
                    # grid step of this token's groups bounds the dequantization error
                    for g in range(4):
                        sg = x[32 * g:32 * g + 32]
                        step = (sg.max() - sg.min()) / (2 ** L.k_bits[sec] - 1)
                        assert np.all(np.abs(kh[32 * g:32 * g + 32] - sg) <= 0.5 * step * 1.01 + 1e-6)
    assert c.seq_len.tolist() == [105, 1, 266]
    assert int(c.ring_ptr[0]) == int(c.pages.sum())
