"""Pins of the oracle's attention (Eq. 1 over the dequantized cache) and split merge.

Independent anchors: numpy softmax attention over the ORIGINAL fp16 keys and
values of caches whose groups lie exactly on the quantization grid (so the
cache loses nothing); exact special cases (one token, identical keys, empty
head); pruned tokens contributing nothing; the error bound of an all-high,
unpruned cache against uncompressed attention; associativity of the
sequence-split merge (Sec. 6.2).
"""
import numpy as np
import pytest

D = 128


def _np_attention(q, K, V, scale):
    """Textbook softmax attention in fp64 (Eq. 1, one query)."""
    lg = scale * (K @ q)
    w = np.exp(lg - lg.max())
    return (w[:, None] * V).sum(0) / w.sum(), lg.max() + np.log(w.sum())


def _grid_vector(rng, bits, scale_exp_range=(-6, -1)):
    """A D-vector whose every 32-group is z + s*c exactly, s a power of two, both end codes used."""
    lb = (1 << bits) - 1
    out = np.empty(D)
    for g in range(D // 32):
        s = 2.0 ** int(rng.integers(*scale_exp_range))
        z = float(rng.integers(-20, 20)) * s
        c = rng.integers(0, lb + 1, 32)
        i0, i1 = rng.choice(32, 2, replace=False)
        c[i0], c[i1] = 0, lb
        out[32 * g:32 * g + 32] = z + s * c
    assert np.array_equal(out.astype(np.float16).astype(np.float64), out)
    return out


def _build(orc, rng, B, Hkv, n, nh, nl, kv_bits=((8, 4), (4, 2)), window=0, grid=True,
           tokens=(16, 32)):
    """Cache where the top-nh scores are high, next nl low (quota form)."""
    L = orc.layout(k_bits=(kv_bits[0][0], kv_bits[1][0]), v_bits=(kv_bits[0][1], kv_bits[1][1]),
                   tokens_per_page=tokens, max_seq_len=max(n, 1))
    score = np.stack([rng.permutation(B * n).reshape(B, n)[:, :] for _ in range(Hkv)], -1)
    score = score.reshape(B * n, Hkv).astype(np.float32)
    k = np.empty((B * n, Hkv, D))
    v = np.empty((B * n, Hkv, D))
    for b in range(B):
        for h in range(Hkv):
            sc = score[b * n:(b + 1) * n, h]
            order = np.argsort(-sc, kind="stable")
            for r, j in enumerate(order):
                sec = 0 if r < nh else 1
                if grid:
                    k[b * n + j, h] = _grid_vector(rng, L.k_bits[sec])
                    v[b * n + j, h] = _grid_vector(rng, L.v_bits[sec])
                else:
                    k[b * n + j, h] = rng.standard_normal(D)
                    v[b * n + j, h] = rng.standard_normal(D)
    c = orc.Cache(L, B * Hkv * (n // tokens[0] + 3), B, Hkv,
                  ring=rng.permutation(B * Hkv * (n // tokens[0] + 3)))
    quota = np.zeros((B, Hkv, 2), np.int32)
    quota[..., 0], quota[..., 1] = nh, nl
    kb = k.astype(np.float16).view(np.uint16)
    vb = v.astype(np.float16).view(np.uint16)
    orc.quantize_append(c, np.full(B, n, np.int32), kb, vb, score, quota=quota, window=window)
    assert c.status[0] == 0
    return L, c, k.astype(np.float16).astype(np.float64), v.astype(np.float16).astype(np.float64), score


@pytest.mark.parametrize("g", [1, 2, 3])
def test_grid_exact_cache_equals_uncompressed_attention(orc, g):
    rng = np.random.default_rng(40 + g)
    B, Hkv, n, nh, nl = 2, 2, 90, 35, 40
    L, c, k, v, score = _build(orc, rng, B, Hkv, n, nh, nl)
    Hq = Hkv * g
    q = rng.standard_normal((B, Hq, D)).astype(np.float16).view(np.uint16)
    scale = 1.0 / np.sqrt(D)
    out, lse = orc.attention(c, q, scale)
    for b in range(B):
        for hq in range(Hq):
            h = hq // g
            sc = score[b * n:(b + 1) * n, h]
            kept = np.argsort(-sc, kind="stable")[:nh + nl]
            qv = q[b, hq].view(np.float16).astype(np.float64)
            ref, ref_lse = _np_attention(qv, k[b * n + kept, h], v[b * n + kept, h], scale)
            assert np.allclose(out[b, hq], ref, rtol=1e-12, atol=1e-12)
            assert lse[b, hq] == pytest.approx(ref_lse, rel=1e-12)


def test_single_token_and_identical_keys(orc):
    rng = np.random.default_rng(50)
    L, c, k, v, score = _build(orc, rng, 1, 1, 5, 1, 0, grid=False)
    q = rng.standard_normal((1, 1, D)).astype(np.float16).view(np.uint16)
    out, lse = orc.attention(c, q, 0.3)
    kh, vh, _, _ = orc.read_token(c, 0, 0, 0)
    assert np.array_equal(out[0, 0], vh)
    qv = q[0, 0].view(np.float16).astype(np.float64)
    assert lse[0, 0] == pytest.approx(0.3 * qv @ kh, rel=1e-14)
    # identical keys (same precision, so the same dequantized key): uniform weights ->
    # mean of the dequantized values
    n = 40
    kk = np.repeat(rng.standard_normal((1, 1, D)), n, 0).astype(np.float16).view(np.uint16)
    vv = rng.standard_normal((n, 1, D)).astype(np.float16).view(np.uint16)
    L = orc.layout(max_seq_len=n)
    c = orc.Cache(L, 8, 1, 1)
    orc.quantize_append(c, np.array([n]), kk, vv, rng.random((n, 1)).astype(np.float32),
                        quota=np.array([[[n, 0]]]))
    out, _ = orc.attention(c, q, 0.3)
    vh = [orc.read_token(c, 0, 0, u)[1] for u in range(n)]
    assert np.allclose(out[0, 0], np.mean(vh, 0), rtol=0, atol=1e-13)


def test_pruned_tokens_contribute_nothing(orc):
    rng = np.random.default_rng(51)
    n, H = 100, 2
    L = orc.layout(max_seq_len=n)
    k = rng.standard_normal((n, H, D)).astype(np.float16).view(np.uint16)
    v = rng.standard_normal((n, H, D)).astype(np.float16).view(np.uint16)
    score = rng.random((n, H)).astype(np.float32)
    quota = np.array([[[30, 30], [10, 50]]], np.int32)
    outs = []
    for trial in range(2):
        kk, vv = k.copy(), v.copy()
        if trial:
            for h in range(H):
                cls = orc.classify(score[:, h], quota=quota[0, h])
                pr = np.where(cls < 0)[0]
                kk[pr, h] = (rng.standard_normal((len(pr), D)) * 100).astype(np.float16).view(np.uint16)
                vv[pr, h] = (rng.standard_normal((len(pr), D)) * 100).astype(np.float16).view(np.uint16)
        c = orc.Cache(L, 16, 1, H)
        orc.quantize_append(c, np.array([n]), kk, vv, score, quota=quota)
        q = np.random.default_rng(9).standard_normal((1, 4, D)).astype(np.float16).view(np.uint16)
        outs.append(orc.attention(c, q, 0.1))
    assert np.array_equal(outs[0][0], outs[1][0]) and np.array_equal(outs[0][1], outs[1][1])


def test_all_high_cache_approaches_uncompressed(orc):
    """No pruning, all tokens high: error within the perturbation bound, shrinking with bits."""
    rng = np.random.default_rng(52)
    n = 64
    errs = []
    for kb, vb in [(4, 2), (8, 4), (8, 8)]:
        L = orc.layout(k_bits=(kb, kb), v_bits=(vb, vb), tokens_per_page=(16, 16), max_seq_len=n)
        k = rng.standard_normal((n, 1, D)).astype(np.float16)
        v = rng.standard_normal((n, 1, D)).astype(np.float16)
        c = orc.Cache(L, 8, 1, 1)
        orc.quantize_append(c, np.array([n]), k.view(np.uint16), v.view(np.uint16),
                            rng.random((n, 1)).astype(np.float32), quota=np.array([[[n, 0]]]))
        q = rng.standard_normal((1, 1, D)).astype(np.float16)
        scale = 1.0 / np.sqrt(D)
        out, _ = orc.attention(c, q.view(np.uint16), scale)
        K = k[:, 0].astype(np.float64)
        V = v[:, 0].astype(np.float64)
        ref, _ = _np_attention(q[0, 0].astype(np.float64), K, V, scale)
        Kh = np.array([orc.read_token(c, 0, 0, u)[0] for u in range(n)])
        Vh = np.array([orc.read_token(c, 0, 0, u)[1] for u in range(n)])
        dk, dv = np.abs(Kh - K).max(), np.abs(Vh - V).max()
        delta = scale * np.abs(q[0, 0].astype(np.float64)).sum() * dk
        bound = (np.exp(2 * delta) - 1) * np.abs(V).max() + dv
        err = np.abs(out[0, 0] - ref).max()
        assert err <= bound
        errs.append(err)
    assert errs[0] > errs[1] > errs[2]


def test_split_merge_is_associative(orc):
    rng = np.random.default_rng(53)
    L, c, k, v, score = _build(orc, rng, 1, 2, 300, 100, 150, grid=False)
    q = rng.standard_normal((1, 4, D)).astype(np.float16).view(np.uint16)
    out, lse = orc.attention(c, q, 0.08)
    for hq in range(4):
        t = hq // 2
        P = int(c.pages[t].sum())
        for trial in range(5):
            cuts = np.sort(rng.choice(np.arange(1, P), size=int(rng.integers(1, min(6, P))), replace=False))
            bounds = [0] + cuts.tolist() + [P]
            if trial == 0:
                bounds = [0, 0, P, P]  # empty splits carry m = -inf
            parts = [orc.attention_partial(c, q, 0.08, 0, hq, a, b) for a, b in zip(bounds, bounds[1:])]
            m = np.array([p[0] for p in parts])
            l = np.array([p[1] for p in parts])
            acc = np.stack([p[2] for p in parts])
            o, ls = orc.merge_partials(m, l, acc)
            assert np.allclose(o, out[0, hq], rtol=1e-12, atol=1e-13)
            assert ls == pytest.approx(lse[0, hq], rel=1e-13)


def test_empty_head(orc):
    L = orc.layout(max_seq_len=64)
    c = orc.Cache(L, 8, 2, 1)
    rng = np.random.default_rng(54)
    k = rng.standard_normal((10, 1, D)).astype(np.float16).view(np.uint16)
    orc.quantize_append(c, np.array([10, 0]), k, k, rng.random((10, 1)).astype(np.float32),
                        quota=np.array([[[5, 0]], [[0, 0]]]))
    q = rng.standard_normal((2, 1, D)).astype(np.float16).view(np.uint16)
    out, lse = orc.attention(c, q, 0.1)
    assert np.all(out[1] == 0) and lse[1, 0] == -np.inf
    assert np.isfinite(lse[0, 0])
    o, ls = orc.merge_partials(np.array([-np.inf]), np.array([0.0]), np.zeros((1, D)))
    assert np.all(o == 0) and ls == -np.inf
