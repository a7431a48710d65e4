"""Pins of the oracle's generation-phase policy (Sec. 4, Algorithm 1), CPU only.

Worked cases, one per branch of Algorithm 1, whose outcomes are derived by hand
from the scores they set; then invariants of random multi-step runs (window
tokens stay high, tokens only move high -> low, sections stay dense, unused
slots stay zero, untouched tokens keep their bytes, re-quantization error
bounds, page and ring accounting).
"""
import numpy as np
import pytest

ALPHA_H, ALPHA_L = 0.9, 0.45   # with N = 9: thresholds 0.1 and 0.05
W = 2


def _sections(orc, c, t):
    out = {}
    for sec in (0, 1):
        toks = {}
        for u in range(int(c.len[t, sec])):
            kh, vh, s, pos = orc.read_token(c, t, sec, u)
            assert pos not in toks
            toks[pos] = (s, kh, vh)
        out[sec] = toks
    return out


def _prompt_then_decode(orc, prompt_scores, cand_score, seed=3):
    """One table: 8 prompt tokens (positions 0..7, window W = 2, quota (2, 2) over
    positions 0..5), then one decode token (position 8, high)."""
    rng = np.random.default_rng(seed)
    L = orc.layout(max_seq_len=64)
    c = orc.Cache(L, 16, 1, 1, ring=np.arange(16))
    score = np.array(list(prompt_scores) + [cand_score, 0.5], np.float32).reshape(8, 1)
    k = rng.standard_normal((8, 1, 128)).astype(np.float16).view(np.uint16)
    v = rng.standard_normal((8, 1, 128)).astype(np.float16).view(np.uint16)
    orc.quantize_append(c, np.array([8], np.int32), k, v, score,
                        quota=np.array([[[2, 2]]], np.int32), window=W)
    kd = rng.standard_normal((1, 1, 128)).astype(np.float16).view(np.uint16)
    vd = rng.standard_normal((1, 1, 128)).astype(np.float16).view(np.uint16)
    orc.quantize_append(c, np.array([1], np.int32), kd, vd, np.array([[0.3]], np.float32),
                        quota=np.array([[[1, 0]]], np.int32))
    assert int(c.seq_len[0]) == 9 and int(c.status[0]) == 0
    return c


@pytest.mark.parametrize("prompt,cand,high,low", [
    # t_c stays high; the high victim (position 0, 0.08) is in [0.05, 0.1): moves low
    ([0.08, 0.09, 0.07, 0.06, 0.01, 0.02], 0.5, {1, 6, 7, 8}, {0, 2, 3}),
    # t_c stays high; the high victim (position 0, 0.03) is below 0.05: removed
    ([0.03, 0.04, 0.02, 0.015, 0.01, 0.005], 0.5, {1, 6, 7, 8}, {2, 3}),
    # t_c stays high; the high victim (position 0, 0.3) stays
    ([0.3, 0.4, 0.2, 0.06, 0.01, 0.02], 0.5, {0, 1, 6, 7, 8}, {2, 3}),
    # t_c (0.07) moves low; the low victim (position 3, 0.01) is evicted
    ([0.3, 0.4, 0.2, 0.01, 0.005, 0.002], 0.07, {0, 1, 7, 8}, {2, 6}),
    # t_c (0.07) moves low; the low victim (position 3, 0.06) stays
    ([0.3, 0.4, 0.2, 0.06, 0.005, 0.002], 0.07, {0, 1, 7, 8}, {2, 3, 6}),
    # t_c (0.01) is removed
    ([0.3, 0.4, 0.2, 0.06, 0.005, 0.002], 0.01, {0, 1, 7, 8}, {2, 3}),
    # equal lowest high scores (positions 0 and 1, 0.08): the lower position moves
    ([0.08, 0.08, 0.07, 0.06, 0.01, 0.02], 0.5, {1, 6, 7, 8}, {0, 2, 3}),
])
def test_algorithm1_branches(orc, prompt, cand, high, low):
    c = _prompt_then_decode(orc, prompt, cand)
    before = _sections(orc, c, 0)
    orc.generation_step(c, ALPHA_H, ALPHA_L, W)
    assert int(c.status[0]) == 0
    after = _sections(orc, c, 0)
    assert set(after[0]) == high and set(after[1]) == low
    for sec in (0, 1):
        for pos, (s, kh, vh) in after[sec].items():
            if pos in before[sec]:          # untouched: same values, same score
                s0, k0, v0 = before[sec][pos]
                assert s == s0 and np.array_equal(kh, k0) and np.array_equal(vh, v0)
            else:                           # moved high -> low: re-quantized
                assert sec == 1 and pos in before[0]
                s0, k0, v0 = before[0][pos]
                assert s == s0
                _assert_requant_close(k0, kh, 4)
                _assert_requant_close(v0, vh, 2)


def _assert_requant_close(x, y, bits):
    """Low-precision codes of the high token's fp16 values: within half a low
    quantization step of the group's range (plus fp16 rounding) per element."""
    for g in range(4):
        xs, ys = x[32 * g:32 * g + 32], y[32 * g:32 * g + 32]
        step = (xs.max() - xs.min()) / (2 ** bits - 1)
        tol = 0.5 * step * (1 + 2 ** -9) + 2 ** -10 * max(1.0, np.abs(xs).max())
        assert np.abs(xs - ys).max() <= tol


def test_no_candidate_no_change(orc):
    """N - 1 - W < 0, or the candidate position not held high: nothing changes."""
    c = _prompt_then_decode(orc, [0.3, 0.4, 0.2, 0.06, 0.005, 0.002], 0.01)
    snap = c.copy()
    orc.generation_step(c, ALPHA_H, ALPHA_L, 20)   # window longer than the sequence
    for f in ("pool", "table", "pages", "len", "seq_len", "ring", "ring_ptr", "status"):
        assert np.array_equal(getattr(c, f), getattr(snap, f))
    orc.generation_step(c, ALPHA_H, ALPHA_L, 4)    # position 4 was pruned by the prompt
    for f in ("pool", "table", "pages", "len", "ring_ptr"):
        assert np.array_equal(getattr(c, f), getattr(snap, f))


def _unused_slots_zero(orc, c, t):
    L = c.L
    for sec in (0, 1):
        T = L.tokens_per_page[sec]
        n, npg = int(c.len[t, sec]), int(c.pages[t, sec])
        for pi in range(npg):
            slot = c.table[t, pi] if sec == 0 else c.table[t, L.p_max - 1 - pi]
            pg = c.pool[slot]
            kb, vb = L.k_bits[sec], L.v_bits[sec]
            for s in range(T):
                if pi * T + s < n:
                    continue
                for ch in range(128 * kb // 128):
                    o = L.off_kcode[sec] + (ch * T + s) * 16
                    assert not pg[o:o + 16].any()
                assert not pg[L.off_kmeta[sec] + s * 16:L.off_kmeta[sec] + s * 16 + 16].any()
                rows = pg[L.off_vcode[sec]:L.off_vcode[sec] + 128 * T * vb // 8].reshape(128, -1)
                bits = np.unpackbits(rows, axis=1, bitorder="little")
                assert not bits[:, s * vb:(s + 1) * vb].any()
                for g in range(4):
                    o = L.off_vmeta[sec] + (g * T + s) * 4
                    assert not pg[o:o + 4].any()
                assert not pg[L.off_score[sec] + 4 * s:L.off_score[sec] + 4 * s + 4].any()
                assert not pg[L.off_pos[sec] + 4 * s:L.off_pos[sec] + 4 * s + 4].any()


def test_random_steps_invariants(orc):
    """Two sequences x two KV heads, threshold-form prompt with a window, then
    decode steps of append + policy; every step's change checked."""
    rng = np.random.default_rng(31)
    B, H, Wn = 2, 2, 8
    L = orc.layout(max_seq_len=400)
    c = orc.Cache(L, 200, B, H, ring=rng.permutation(200))
    n0 = np.array([150, 90], np.int32)
    rows = int(n0.sum())
    k = rng.standard_normal((rows, H, 128)).astype(np.float16).view(np.uint16)
    v = rng.standard_normal((rows, H, 128)).astype(np.float16).view(np.uint16)
    sc = (rng.random((rows, H)) ** 3 * 0.05).astype(np.float32)
    ah, al = 1.0, 0.3
    orc.quantize_append(c, n0, k, v, sc, alpha_h=ah, alpha_l=al, window=Wn)
    moved = removed = 0
    for step in range(40):
        kd = rng.standard_normal((B, H, 128)).astype(np.float16).view(np.uint16)
        vd = rng.standard_normal((B, H, 128)).astype(np.float16).view(np.uint16)
        sd = (rng.random((B, H)) ** 3 * 0.05).astype(np.float32)
        orc.quantize_append(c, np.ones(B, np.int32), kd, vd, sd,
                            quota=np.tile(np.array([1, 0], np.int32), (B, H, 1)))
        before = [_sections(orc, c, t) for t in range(B * H)]
        pages0, head0 = c.pages.copy(), int(c.ring_ptr[0])
        orc.generation_step(c, ah, al, Wn)
        assert int(c.status[0]) == 0
        grew = 0
        for t in range(B * H):
            N = int(c.seq_len[t // H])
            after = _sections(orc, c, t)
            hb, lb = set(before[t][0]), set(before[t][1])
            ha, la = set(after[0]), set(after[1])
            # window positions all high, before and after
            win = set(range(N - Wn, N))
            assert win <= hb and win <= ha
            # only high -> low moves, at most one token leaves high, at most one leaves low
            assert ha <= hb and la <= lb | hb
            assert len(hb - ha) <= 1 and len(lb - la) <= 1
            gone = (hb | lb) - (ha | la)
            moved += len(la - lb)
            removed += len(gone)
            assert len(la - lb) + len(gone) <= 2
            # untouched tokens keep their values; moved ones keep score and position
            for sec in (0, 1):
                for pos, (s, kh, vh) in after[sec].items():
                    src = before[t][sec].get(pos)
                    if src is not None:
                        assert s == src[0] and np.array_equal(kh, src[1]) and np.array_equal(vh, src[2])
                    else:
                        assert before[t][0][pos][0] == s
            # dense sections, unused slots zero, at most one new low page
            for sec in (0, 1):
                T = L.tokens_per_page[sec]
                assert c.len[t, sec] <= c.pages[t, sec] * T
            assert c.pages[t, 0] == pages0[t, 0]
            assert 0 <= c.pages[t, 1] - pages0[t, 1] <= 1
            grew += int(c.pages[t, 1] - pages0[t, 1])
            _unused_slots_zero(orc, c, t)
        assert int(c.ring_ptr[0]) - head0 == grew
    assert moved > 0 and removed > 0   # both kinds of change happened


def test_out_of_pages_changes_nothing(orc):
    """A candidate that must go to a full low section when the ring is empty:
    status OUT_OF_PAGES, state unchanged.  Prompt of 40 (window 2, quota (2, 32)
    over positions 0..37: one full low page), one decode token, N = 41."""
    rng = np.random.default_rng(5)
    L = orc.layout(max_seq_len=128)
    c = orc.Cache(L, 16, 1, 1, ring=np.arange(16))
    sc = np.concatenate([[0.5, 0.4], np.linspace(0.06, 0.09, 32), [0.001] * 4,
                         [0.07, 0.5]]).astype(np.float32).reshape(40, 1)
    k = rng.standard_normal((40, 1, 128)).astype(np.float16).view(np.uint16)
    v = rng.standard_normal((40, 1, 128)).astype(np.float16).view(np.uint16)
    orc.quantize_append(c, np.array([40], np.int32), k, v, sc,
                        quota=np.array([[[2, 32]]], np.int32), window=2)
    orc.quantize_append(c, np.array([1], np.int32), k[:1], v[:1], np.array([[0.3]], np.float32),
                        quota=np.array([[[1, 0]]], np.int32))
    assert c.len[0, 1] == 32 and c.pages[0, 1] == 1 and int(c.seq_len[0]) == 41
    ah, al = 4.1, 2.05   # thresholds 0.1 and 0.05 at N = 41
    c.ring_ptr[0] = c.ring_ptr[1]   # no free page
    snap = c.copy()
    orc.generation_step(c, ah, al, 2)
    assert int(c.status[0]) & 1
    for f in ("pool", "table", "pages", "len", "ring_ptr"):
        assert np.array_equal(getattr(c, f), getattr(snap, f))
    # with a free page the same step moves position 38 to a new low page
    c2 = snap.copy()
    c2.status[:] = 0
    c2.ring_ptr[0] = c2.ring_ptr[1] - 1
    orc.generation_step(c2, ah, al, 2)
    assert int(c2.status[0]) == 0 and c2.len[0, 1] == 33 and c2.pages[0, 1] == 2
    assert orc.read_token(c2, 0, 1, 32)[3] == 38


def test_requantization_rounding_hand_worked(orc):
    """Re-quantization of a high token to low precision, worked by hand: each element
    is s*code + z as one fp32 fma, rounded to fp16 (nearest even), then quantized as a
    low-precision token.  The case is built so that this exact order decides a low
    code: the product of an fp16 scale and an integer code of at most 8 bits is exact
    in fp32, so s*c lands exactly on an fp16 midpoint, and z = -2^-24 (fp16 0x8001)
    sits below fp32's half-ulp there.  fp32 rounding therefore returns the midpoint
    and the fp16 rounding takes the even neighbour above it, while skipping the fp16
    rounding keeps the midpoint and rounding the exact value once goes to the odd
    neighbour below.  (A separate multiply then add gives the fma's result here,
    since the product is exact.)

    Key group 0 (K8 -> K4), s = 0x3C01 = 1 + 2^-10, z = -2^-24, codes 0, 3, 6 then 0:
      3s = 3 + 1.5*2^-9: midpoint of 3 + 2^-9 (odd) and 3 + 2^-8 (even) -> 3.00390625
      6s = 6 + 1.5*2^-8: midpoint of 6 + 2^-8 (odd) and 6 + 2^-7 (even) -> 6.0078125
      min = -2^-24, max = 6.0078125 (adding 2^-24 is lost in fp32),
      s_lo = fp16(6.0078125 / 15 = 0.4005208) = 1641 * 2^-12 = 0.400634765625 (0x3669),
      codes: 3.00390625 / 0.400634765625 = 7.498 -> 7; 6.0078125 / s_lo = 14.996 -> 15.
      Without the fp16 rounding: s_lo = 0.400390625, 3.0029296875 / s_lo = 7.5 -> 8.
      With one rounding of the exact value: 3.001953125 / 0.400146484375 = 7.502 -> 8.
    Value group 0 (V4 -> V2), s = 0x3C16 = 1.021484375, z = -2^-24, codes 0, 5, 6 then 0:
      5s = 5.107421875 = 1307.5 * 2^-8: midpoint -> 1308 * 2^-8 = 5.109375 (even)
      6s = 6.12890625 (exact in fp16), s_lo = 6.12890625 / 3 = 2.04296875 (0x4016),
      code 5.109375 / 2.04296875 = 2.5010 -> 3.
      Without the fp16 rounding: 5.107421875 / 2.04296875 = 2.5 -> 2 (even);
      with one rounding of the exact value: 5.10546875 / 2.04296875 = 2.4990 -> 2.
    """
    c = _prompt_then_decode(orc, [0.08, 0.09, 0.07, 0.06, 0.01, 0.02], 0.5)
    L = c.L
    assert orc.read_token(c, 0, 0, 0)[3] == 0    # high index 0 holds position 0, the victim
    pg = c.pool[int(c.table[0, 0])]              # its page; slot 0
    kc = np.zeros(32, np.uint8)
    kc[1:3] = [3, 6]
    for d in range(32):                          # K8 chunk d // 16, byte d % 16 of slot 0
        pg[L.off_kcode[0] + (d // 16) * 16 * 16 + d % 16] = kc[d]
    pg[L.off_kmeta[0]:L.off_kmeta[0] + 4] = np.array([0x3C01, 0x8001], np.uint16).view(np.uint8)
    vc = np.zeros(32, np.uint8)
    vc[1:3] = [5, 6]
    for d in range(32):                          # V4 row d: slot 0 in the low nibble of byte 0
        o = L.off_vcode[0] + d * 8
        pg[o] = (pg[o] & 0xF0) | vc[d]
    pg[L.off_vmeta[0]:L.off_vmeta[0] + 4] = np.array([0x3C16, 0x8001], np.uint16).view(np.uint8)
    orc.generation_step(c, ALPHA_H, ALPHA_L, W)
    assert int(c.status[0]) == 0
    u = [orc.read_token(c, 0, 1, i)[3] for i in range(int(c.len[0, 1]))].index(0)
    lp = c.pool[int(c.table[0, L.p_max - 1 - u // 32])]
    s = u % 32
    kcodes = [(lp[L.off_kcode[1] + s * 16 + d // 2] >> (4 * (d % 2))) & 15 for d in range(32)]
    vcodes = [(lp[L.off_vcode[1] + d * 8 + s // 4] >> (2 * (s % 4))) & 3 for d in range(32)]
    kmeta = lp[L.off_kmeta[1] + s * 16:L.off_kmeta[1] + s * 16 + 4].view(np.uint16)
    vmeta = lp[L.off_vmeta[1] + s * 4:L.off_vmeta[1] + s * 4 + 4].view(np.uint16)
    assert kcodes == [0, 7, 15] + [0] * 29
    assert kmeta.tolist() == [0x3669, 0x8001]
    assert vcodes == [0, 3, 3] + [0] * 29
    assert vmeta.tolist() == [0x4016, 0x8001]
