"""Pins of the oracle's significance update (Sec. 4: a token's significance is the mean
of the attention scores it receives, the scores of a KV head's query heads combined by
their maximum), one decode step at a time.

Independent anchors:
  - grid-exact caches (groups exactly on the quantization grid, so the cache holds the
    original fp16 keys): the expected probabilities come from numpy softmax over the
    original keys and the scores/positions as appended, without any oracle read-back;
  - closed forms: a table keeping one token gives it probability 1; the newest token
    (count 1) takes its probability as score; with one head per KV head the
    probabilities of a table sum to one; k decode steps equal the plain mean of the
    k + c0 received values;
  - pruned tokens are not scored (the kept ones see a softmax over kept tokens only).
"""
import numpy as np
import pytest

from test_oracle_attention import D, _grid_vector

SCALE = 1.0 / np.sqrt(D)


def _grid_both(rng):
    """A key vector exact at both 8 and 4 bits: every 32-group is z + 17 * 2^e * c with
    c in 0..15, both end codes used (the 8-bit scale is 2^e, the 4-bit one 17 * 2^e)."""
    out = np.empty(D)
    for g in range(D // 32):
        e = int(rng.integers(-8, -3))
        z = float(rng.integers(-300, 300)) * 2.0 ** e
        c = rng.integers(0, 16, 32)
        i0, i1 = rng.choice(32, 2, replace=False)
        c[i0], c[i1] = 0, 15
        out[32 * g:32 * g + 32] = z + 17.0 * 2.0 ** e * c
    assert np.array_equal(out.astype(np.float16).astype(np.float64), out)
    return out


def _grid_cache(orc, rng, B, Hkv, n, quota, score=None):
    L = orc.layout(max_seq_len=n + 8)
    k = np.stack([[_grid_both(rng) for _ in range(Hkv)] for _ in range(B * n)])
    v = rng.standard_normal((B * n, Hkv, D)).astype(np.float16)
    if score is None:
        score = rng.random((B * n, Hkv)).astype(np.float32) * np.float32(0.01)
    npg = B * Hkv * (n // 16 + 4)
    c = orc.Cache(L, npg, B, Hkv, ring=rng.permutation(npg))
    orc.quantize_append(c, np.full(B, n, np.int32), k.astype(np.float16).view(np.uint16),
                        v.view(np.uint16), score, quota=np.asarray(quota, np.int32))
    assert c.status[0] == 0
    return c, k, score


def _kept(orc, c, t):
    """(section, index, score, position) of every kept token of table t, section order."""
    out = []
    for sec in (0, 1):
        for u in range(int(c.len[t, sec])):
            _, _, s, p = orc.read_token(c, t, sec, u)
            out.append((sec, u, float(s), int(p)))
    return out


@pytest.mark.parametrize("g", [1, 3, 4])
def test_grid_exact_against_numpy_softmax(orc, g):
    """Every kept token's new score against numpy: probabilities from the original
    keys of the kept positions, max over the g heads, running mean over N - p."""
    rng = np.random.default_rng(80 + g)
    B, Hkv, n = 2, 2, 70
    quota = np.tile(np.array([20, 25], np.int32), (B, Hkv, 1))   # 25 tokens pruned per table
    c, k, score = _grid_cache(orc, rng, B, Hkv, n, quota)
    before = {t: _kept(orc, c, t) for t in range(B * Hkv)}
    q = rng.standard_normal((B, Hkv * g, D)).astype(np.float16)
    orc.update_significance(c, q.view(np.uint16), SCALE)
    N = n
    for b in range(B):
        for h in range(Hkv):
            t = b * Hkv + h
            pos = np.array([p for _, _, _, p in before[t]])
            assert len(pos) == 45
            K = k[b * n + pos, h].astype(np.float64)          # original keys, as appended
            x = np.zeros(len(pos))
            for hq in range(h * g, (h + 1) * g):
                lg = SCALE * (K @ q[b, hq].astype(np.float64))
                p = np.exp(lg - lg.max())
                x = np.maximum(x, p / p.sum())
            s0 = score[b * n + pos, h].astype(np.float64)       # the appended scores
            want = (s0 + (x - s0) / (N - pos)).astype(np.float32)
            got = np.array([s for _, _, s, _ in _kept(orc, c, t)], np.float32)
            assert np.allclose(got, want, rtol=2e-6, atol=1e-9), (b, h)


def test_single_kept_token_and_newest_token(orc):
    """A table keeping one token: its probability is 1.  The newest token (position
    N - 1, count 1) takes x itself as its score, whatever it held."""
    rng = np.random.default_rng(90)
    n = 33
    score = rng.random((n, 2)).astype(np.float32)
    score[n - 1, :] = 5.0                                  # the newest token is kept high
    quota = np.array([[[1, 0], [3, 4]]], np.int32)         # table 0 keeps one token
    c, k, _ = _grid_cache(orc, rng, 1, 2, n, quota, score=score)
    q = rng.standard_normal((1, 2, D)).astype(np.float16).view(np.uint16)
    orc.update_significance(c, q, SCALE)
    (sec, u, s, p), = _kept(orc, c, 0)
    assert p == n - 1 and s == np.float32(1.0)
    kept1 = _kept(orc, c, 1)
    newest = [s for _, _, s, p in kept1 if p == n - 1]
    assert len(newest) == 1 and 0.0 < newest[0] <= 1.0


def test_probabilities_sum_to_one_with_one_head_per_kv_head(orc):
    """g = 1: x is the head's softmax over the table's kept tokens, so
    sum_j [(s_new - s_old) * (N - p) + s_old] = sum_j x_j = 1."""
    rng = np.random.default_rng(91)
    n = 200
    quota = np.array([[[60, 80]]], np.int32)
    c, k, score = _grid_cache(orc, rng, 1, 1, n, quota)
    old = _kept(orc, c, 0)
    q = (rng.standard_normal((1, 1, D)) * 3).astype(np.float16).view(np.uint16)
    orc.update_significance(c, q, SCALE)
    new = _kept(orc, c, 0)
    xs = [(sn - so) * (n - p) + so for (_, _, so, p), (_, _, sn, _) in zip(old, new)]
    assert abs(sum(xs) - 1.0) < 1e-4


def test_running_mean_over_steps(orc):
    """Three decode steps, each appending one high token and updating: a prompt token
    at position p ends with (c0 * s0 + x1 + x2 + x3) / (c0 + 3), c0 = n - p, the x_i
    from numpy over the tokens kept at each step."""
    rng = np.random.default_rng(92)
    n = 50
    quota = np.array([[[30, 0]]], np.int32)
    c, k, score = _grid_cache(orc, rng, 1, 1, n, quota)
    c.seq_len[0] = n
    track = {p: float(s) for _, _, s, p in _kept(orc, c, 0)}   # appended scores (positions < n)
    keys = {p: k[p, 0].astype(np.float64) for p in track}
    xs = {p: [] for p in track}
    for step in range(3):
        kd = _grid_vector(rng, 8)
        orc.quantize_append(c, np.array([1], np.int32), kd.astype(np.float16).view(np.uint16)[None, None],
                            rng.standard_normal((1, 1, D)).astype(np.float16).view(np.uint16),
                            np.array([[0.5]], np.float32), quota=np.array([[[1, 0]]], np.int32))
        keys[n + step] = kd
        q = rng.standard_normal((1, 1, D)).astype(np.float16)
        pos = sorted(keys)
        lg = SCALE * np.array([keys[p] @ q[0, 0].astype(np.float64) for p in pos])
        pr = np.exp(lg - lg.max())
        pr /= pr.sum()
        for p, x in zip(pos, pr):
            if p in xs:
                xs[p].append(x)
        orc.update_significance(c, q.view(np.uint16), SCALE)
    final = {p: s for _, _, s, p in _kept(orc, c, 0)}
    for p, s0 in track.items():
        c0 = n - p
        want = (c0 * s0 + sum(xs[p])) / (c0 + 3)
        assert abs(final[p] - want) <= 1e-6 * max(1.0, abs(want)), p
