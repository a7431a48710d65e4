"""Pins of the oracle's prompt-phase significance (Sec. 4: token p of an N-token prompt
is scored by the mean of the N - p attention probabilities it receives from the queries
p..N-1 (causal, itself included); a KV head's query heads are combined by their maximum,
per query).

Independent anchors:
  - closed forms: zero queries (or equal keys) give uniform rows 1/(j+1), so the score
    is (H_N - H_p) / (N - p) with H the harmonic numbers; two tokens with a chosen logit
    gap give a logistic probability (pins the scale and the softmax);
  - the max over heads, taken per query: two heads that alternate between a uniform row
    and a row peaked on token 0 give token 0 a score of 1 (the maximum of the per-head
    means would be below 1);
  - invariants: with one head per KV head every query's row sums to one, so
    sum_p score_p (N - p) = N; g identical heads equal one head;
  - the decode-time update continues it: prompt scores over N tokens, one appended token
    and one update step equal the prompt scores over N + 1 tokens (grid-exact keys, so
    the cache holds the prompt's keys exactly);
  - brute force: numpy over the full masked matrix on tiny inputs.
"""
import numpy as np
import pytest

from test_oracle_significance import _grid_both

D = 128
SCALE = 1.0 / np.sqrt(D)


def f16(x):
    return np.asarray(x, np.float16).view(np.uint16)


def harmonic_scores(N):
    H = np.concatenate([[0.0], np.cumsum(1.0 / np.arange(1, N + 1))])
    return np.array([(H[N] - H[p]) / (N - p) for p in range(N)])


def numpy_scores(new_len, q, k, scale):
    """Brute force: per sequence and KV head, the full N x N masked softmax of each query
    head, the elementwise maximum over the group, column means over the N - p rows."""
    q = q.view(np.float16).astype(np.float64)
    k = k.view(np.float16).astype(np.float64)
    Hq, Hkv = q.shape[1], k.shape[1]
    g = Hq // Hkv
    out = np.zeros((q.shape[0], Hkv))
    r0 = 0
    for N in new_len:
        if N == 0:
            continue
        mask = np.tril(np.ones((N, N), bool))
        for h in range(Hkv):
            P = np.zeros((N, N))
            for hq in range(h * g, (h + 1) * g):
                lg = scale * q[r0:r0 + N, hq] @ k[r0:r0 + N, h].T
                lg = np.where(mask, lg, -np.inf)
                e = np.exp(lg - lg.max(axis=1, keepdims=True))
                P = np.maximum(P, e / e.sum(axis=1, keepdims=True))
            out[r0:r0 + N, h] = P.sum(axis=0) / (N - np.arange(N))
        r0 += N
    return out


@pytest.mark.parametrize("g", [1, 3])
def test_uniform_rows_give_harmonic_scores(orc, g):
    rng = np.random.default_rng(200 + g)
    new_len = np.array([1, 2, 9, 40], np.int32)
    n = int(new_len.sum())
    Hkv = 2
    k = f16(rng.standard_normal((n, Hkv, D)))
    q = f16(np.zeros((n, Hkv * g, D)))                       # zero queries: every row uniform
    s = orc.prompt_significance(new_len, q, k, SCALE)
    r0 = 0
    for N in new_len:
        want = harmonic_scores(int(N))
        for h in range(Hkv):
            assert np.allclose(s[r0:r0 + N, h], want, rtol=1e-6, atol=0), (N, h)
        r0 += N
    assert s[0, 0] == np.float32(1.0)                        # a lone token receives probability 1
    # equal keys with random queries: uniform as well
    k2 = f16(np.tile(rng.standard_normal(D), (n, Hkv, 1)))
    q2 = f16(rng.standard_normal((n, Hkv * g, D)))
    s2 = orc.prompt_significance(new_len, q2, k2, SCALE)
    assert np.allclose(s2[-40:, 1], harmonic_scores(40), rtol=1e-6)


def test_two_tokens_logistic(orc):
    """N = 2, one head: query 1 sees logits a (token 0) and b (token 1);
    score_0 = (1 + sigma(a - b)) / 2 and score_1 = sigma(b - a)."""
    k = np.zeros((2, 1, D))
    k[0, 0, 0], k[1, 0, 1] = 2.0, 1.0
    q = np.zeros((2, 1, D))
    q[1, 0, 0], q[1, 0, 1] = 3.0, -1.5                       # a = 6 * scale, b = -1.5 * scale
    s = orc.prompt_significance(np.array([2], np.int32), f16(q), f16(k), SCALE)
    a, b = 6.0 * SCALE, -1.5 * SCALE
    p0 = 1.0 / (1.0 + np.exp(b - a))
    assert np.isclose(s[0, 0], (1 + p0) / 2, rtol=1e-7)
    assert np.isclose(s[1, 0], 1 - p0, rtol=1e-6)
    # without the scale the same inputs would give a different value
    assert not np.isclose(s[1, 0], 1.0 / (1.0 + np.exp(7.5)), rtol=1e-3)


def test_max_over_heads_is_taken_per_query(orc):
    """Two query heads of one KV head.  Token 0's key points along channel 0; the other
    keys are orthogonal to it.  At even positions head A's query is zero (uniform row)
    and head B's is peaked on token 0 (logit ~70 above the rest), at odd positions the
    other way round, so at every query one head gives token 0 probability ~1."""
    N = 30
    rng = np.random.default_rng(210)
    k = np.zeros((N, 1, D))
    k[0, 0, 0] = 8.0
    k[1:, 0, 1:] = rng.standard_normal((N - 1, D - 1)) * 0.01
    q = np.zeros((N, 2, D))
    peak = np.zeros(D)
    peak[0] = 100.0
    q[0::2, 1] = peak
    q[1::2, 0] = peak
    s = orc.prompt_significance(np.array([N], np.int32), f16(q), f16(k), SCALE)[:, 0].astype(np.float64)
    assert abs(s[0] - 1.0) < 1e-6
    # tokens p > 0: the uniform head's 1/(j+1) wins at every query
    assert np.allclose(s[1:], harmonic_scores(N)[1:], rtol=1e-5)
    # the per-head-mean reading would score token 0 well below 1
    H = harmonic_scores(N)
    assert max(np.mean([1.0 if j % 2 else 1.0 / (j + 1) for j in range(N)]), H[0]) < 0.9


def test_rows_sum_to_one_and_identical_heads(orc):
    rng = np.random.default_rng(220)
    new_len = np.array([57, 130], np.int32)
    n = int(new_len.sum())
    k = f16(rng.standard_normal((n, 1, D)) * 2)
    q = f16(rng.standard_normal((n, 1, D)) * 2)
    s = orc.prompt_significance(new_len, q, k, SCALE)[:, 0].astype(np.float64)
    r0 = 0
    for N in new_len:
        tot = np.sum(s[r0:r0 + N] * (N - np.arange(N)))
        assert abs(tot - N) < 1e-4 * N, (N, tot)
        r0 += N
    q4 = np.repeat(q, 4, axis=1)                             # four identical query heads
    s4 = orc.prompt_significance(new_len, q4, k, SCALE)[:, 0]
    assert np.array_equal(s4, s.astype(np.float32))


def test_against_numpy_brute_force(orc):
    rng = np.random.default_rng(230)
    new_len = np.array([5, 0, 33, 17], np.int32)
    n = int(new_len.sum())
    Hkv, g = 2, 4
    k = f16(rng.standard_normal((n, Hkv, D)) * 2)
    q = f16(rng.standard_normal((n, Hkv * g, D)))
    s = orc.prompt_significance(new_len, q, k, SCALE)
    want = numpy_scores(new_len, q, k, SCALE)
    assert np.allclose(s, want, rtol=2e-7, atol=1e-30)
    # select: only table (sequence 2, head 1) is computed
    sel = np.zeros((4, Hkv), bool)
    sel[2, 1] = True
    out = np.full((n, Hkv), -1.0, np.float32)
    orc.prompt_significance(new_len, q, k, SCALE, select=sel, out=out)
    assert np.array_equal(out[5:38, 1], s[5:38, 1])
    assert np.all(out[:5] == -1) and np.all(out[5:38, 0] == -1) and np.all(out[38:] == -1)


def test_decode_update_continues_the_prompt_scores(orc):
    """Prompt scores over N tokens in a cache (all kept, high precision, keys exact at
    8 bits), one appended token and one decode-time update: the kept tokens' scores
    equal the prompt scores over N + 1 tokens."""
    rng = np.random.default_rng(240)
    N, Hkv, g = 45, 2, 3
    keys = np.stack([[_grid_both(rng) for _ in range(Hkv)] for _ in range(N + 1)])
    k = f16(keys)
    q = f16(rng.standard_normal((N + 1, Hkv * g, D)))
    v = f16(rng.standard_normal((N + 1, Hkv, D)))
    s_n = orc.prompt_significance(np.array([N], np.int32), q[:N], k[:N], SCALE)
    s_n1 = orc.prompt_significance(np.array([N + 1], np.int32), q, k, SCALE)
    L = orc.layout(max_seq_len=N + 8)
    c = orc.Cache(L, 32, 1, Hkv, ring=rng.permutation(32))
    orc.quantize_append(c, np.array([N], np.int32), k[:N], v[:N], s_n,
                        quota=np.full((1, Hkv, 2), [N, 0], np.int32))
    orc.quantize_append(c, np.array([1], np.int32), k[N:], v[N:], np.full((1, Hkv), 0.5, np.float32),
                        quota=np.full((1, Hkv, 2), [1, 0], np.int32))
    assert c.status[0] == 0 and c.seq_len[0] == N + 1
    orc.update_significance(c, q[N:N + 1], SCALE)
    for h in range(Hkv):
        got = np.zeros(N + 1)
        for u in range(int(c.len[h, 0])):
            _, _, sc, p = orc.read_token(c, h, 0, u)
            got[p] = sc
        assert np.allclose(got, s_n1[:, h], rtol=2e-6, atol=1e-12), h


def test_tail_equals_the_full_scores(orc):
    """The tail function (only the last m queries) gives the full function's scores of
    the last m tokens, bit for bit after rounding to fp32."""
    rng = np.random.default_rng(250)
    N, Hkv, g = 90, 2, 3
    q = f16(rng.standard_normal((N, Hkv * g, D)))
    k = f16(rng.standard_normal((N, Hkv, D)) * 2)
    full = orc.prompt_significance(np.array([N], np.int32), q, k, SCALE)
    for h in range(Hkv):
        for m in (1, 7, N):
            tail = orc.prompt_significance_tail(q, k, SCALE, h, m)
            assert np.array_equal(tail.astype(np.float32), full[N - m:, h]), (h, m)
    assert orc.prompt_significance_tail(q, k, SCALE, 0, 1)[0] > 0.0
