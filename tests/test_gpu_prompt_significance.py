"""GPU parity of the prompt-phase significance (Sec. 4; diffkv_prompt_significance)
against the oracle: every prompt token's score, the mean of the causal attention
probabilities it receives, maximum over the KV head's query heads per query.

Tolerance: relative 5e-5 (fp32 logits from exact fp16 products and fp32 sums; fp32
row normalizers; the oracle is fp64), absolute 1e-30 (probabilities below 2^-126 may be
flushed to zero on the GPU).  Cases: every group size 1-8 over ragged prompts that span
several query and key blocks with ragged tails; lengths 0, 1 and block multiples;
row normalizers passed in (the row pass skipped); rows cut at total_new; the full
llama8b prompt batch (B=64, Hq=32, Hkv=8, prompts of 1024-4096 tokens) on sampled
tables, plus a row-sum property over every table with one head per KV head; two
32768-token prompts at the long32k head shape on the last tokens of sampled tables.
"""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():  # pragma: no cover
    pytest.skip("needs a GPU", allow_module_level=True)

from oracle import oracle as orc  # noqa: E402
from paper_2412_03131_amd import diffkv as dk  # noqa: E402
from paper_2412_03131_amd import inputs  # noqa: E402

from gpu_util import t  # noqa: E402

D = 128
SCALE = 1.0 / np.sqrt(D)
RTOL, ATOL = 5e-5, 1e-30
LD = dk.layout(max_seq_len=64)   # the call only checks head_dim 128


def _draw(rng, new_len, Hq, Hkv, kscale=2.0):
    n = int(np.sum(new_len))
    q = rng.standard_normal((n, Hq, D)).astype(np.float16).view(np.uint16)
    k = (rng.standard_normal((n, Hkv, D)) * kscale).astype(np.float16).view(np.uint16)
    return q, k


def _close(got, want, what):
    bad = ~(np.abs(got.astype(np.float64) - want) <= RTOL * np.abs(want) + ATOL)
    assert not bad.any(), "%s: %d mismatches, first at %s (gpu %r, oracle %r)" % (
        what, bad.sum(), np.argwhere(bad)[0], got[bad][0], want[bad][0])


def _lse_numpy(new_len, q, k):
    """Natural-log row normalizers of the causal prompt attention (fp64 numpy)."""
    qd = q.view(np.float16).astype(np.float64)
    kd = k.view(np.float16).astype(np.float64)
    Hq, Hkv = q.shape[1], k.shape[1]
    g = Hq // Hkv
    out = np.zeros((q.shape[0], Hq), np.float32)
    r0 = 0
    for N in new_len:
        mask = np.tril(np.ones((N, N), bool))
        for hq in range(Hq):
            lg = SCALE * qd[r0:r0 + N, hq] @ kd[r0:r0 + N, hq // g].T
            lg = np.where(mask, lg, -np.inf)
            m = lg.max(axis=1)
            out[r0:r0 + N, hq] = m + np.log(np.exp(lg - m[:, None]).sum(axis=1))
        r0 += N
    return out


@pytest.mark.parametrize("Hkv,Hq", [(2, 2), (2, 4), (1, 3), (2, 8), (1, 5), (1, 6), (1, 7), (2, 16)])
def test_every_group_size(Hkv, Hq):
    rng = np.random.default_rng(300 + Hq)
    new_len = np.array([1, 17, 64, 65, 300, 0, 257], np.int32)
    q, k = _draw(rng, new_len, Hq, Hkv)
    print("case: prompt significance, group size %d" % (Hq // Hkv), flush=True)
    got = dk.prompt_significance(LD, t(new_len), t(q).view(torch.float16), t(k).view(torch.float16), SCALE)
    torch.cuda.synchronize()
    want = orc.prompt_significance(new_len, q, k, SCALE)
    _close(got.cpu().numpy(), want, "group size %d" % (Hq // Hkv))


def test_given_row_normalizers_and_block_edges():
    """Lengths at and around the block sizes (64 query rows, 256 keys), one long
    sequence; first with the row pass, then with lse passed in."""
    rng = np.random.default_rng(310)
    Hkv, Hq = 2, 8
    new_len = np.array([256, 255, 512, 63, 129, 2], np.int32)
    q, k = _draw(rng, new_len, Hq, Hkv, kscale=3.0)
    want = orc.prompt_significance(new_len, q, k, SCALE)
    qd, kd = t(q).view(torch.float16), t(k).view(torch.float16)
    print("case: prompt significance, block edges", flush=True)
    got = dk.prompt_significance(LD, t(new_len), qd, kd, SCALE)
    torch.cuda.synchronize()
    _close(got.cpu().numpy(), want, "block edges")
    print("case: prompt significance, lse given", flush=True)
    lse = t(_lse_numpy(new_len, q, k))
    got2 = dk.prompt_significance(LD, t(new_len), qd, kd, SCALE, lse=lse)
    torch.cuda.synchronize()
    _close(got2.cpu().numpy(), want, "lse given")


def test_rows_cut_at_total_and_max_new():
    """new_len summing past the rows given: the last sequence is scored over the rows
    that exist; a length above max_new is clamped to it."""
    rng = np.random.default_rng(320)
    Hkv, Hq = 1, 4
    q, k = _draw(rng, [40], Hq, Hkv)
    print("case: prompt significance, rows cut at total_new", flush=True)
    got = dk.prompt_significance(LD, t(np.array([10, 50], np.int32)), t(q).view(torch.float16),
                                 t(k).view(torch.float16), SCALE, max_new=50)
    torch.cuda.synchronize()
    want = orc.prompt_significance(np.array([10, 30], np.int32), q, k, SCALE)
    _close(got.cpu().numpy(), want, "rows cut")
    score = torch.full((40, 1), -1.0, dtype=torch.float32, device="cuda:0")
    dk.prompt_significance(LD, t(np.array([40], np.int32)), t(q).view(torch.float16),
                           t(k).view(torch.float16), SCALE, score=score, max_new=25)
    torch.cuda.synchronize()
    s = score.cpu().numpy()
    want = orc.prompt_significance(np.array([25], np.int32), q[:25], k[:25], SCALE)
    _close(s[:25], want, "clamped to max_new")
    assert np.all(s[25:] == -1.0)


def test_full_llama8b_prompt_batch():
    w = inputs.prefill("llama8b")
    B, Hq, Hkv = w["B"], w["Hq"], w["Hkv"]
    new_len = w["new_len"]
    rows = int(new_len.sum())
    q = inputs.prompt_queries("llama8b", rows)
    print("case: prompt significance, full llama8b (B=%d, rows %d)" % (B, rows), flush=True)
    got = dk.prompt_significance(LD, t(new_len), t(q).view(torch.float16), t(w["k"]).view(torch.float16), SCALE)
    torch.cuda.synchronize()
    g = got.cpu().numpy()
    assert np.all(np.isfinite(g)) and np.all(g >= 0) and np.all(g <= 1.0 + 1e-6)
    sel = np.zeros((B, Hkv), bool)
    b_long = int(np.argmax(new_len))
    sel[b_long, 3] = True
    sel[7, 0] = True
    print("case: oracle on tables (%d, 3) N=%d and (7, 0) N=%d" % (b_long, new_len[b_long], new_len[7]),
          flush=True)
    want = orc.prompt_significance(new_len, q, w["k"], SCALE, select=sel,
                                   out=np.full((rows, Hkv), np.nan, np.float32))
    off = np.concatenate([[0], np.cumsum(new_len)])
    for b, h in np.argwhere(sel):
        r = slice(off[b], off[b + 1])
        _close(g[r, h], want[r, h], "llama8b table (%d, %d)" % (b, h))


def test_row_sums_one_head_per_kv_head_full_size():
    """g = 1 at the llama8b prompt lengths (8 KV heads, one query head each): every query row sums
    to one, so sum_p score_p (N - p) = N for every table."""
    w = inputs.prefill("llama8b")
    new_len = w["new_len"][:16]
    rows = int(new_len.sum())
    rng = np.random.default_rng(330)
    q, k = _draw(rng, new_len, 8, 8)
    print("case: prompt significance, row sums g=1 (rows %d)" % rows, flush=True)
    got = dk.prompt_significance(LD, t(new_len), t(q).view(torch.float16), t(k).view(torch.float16), SCALE)
    torch.cuda.synchronize()
    s = got.cpu().numpy().astype(np.float64)
    off = np.concatenate([[0], np.cumsum(new_len)])
    for b in range(len(new_len)):
        N = int(new_len[b])
        tot = (s[off[b]:off[b + 1]] * (N - np.arange(N))[:, None]).sum(axis=0)
        assert np.allclose(tot, N, rtol=1e-4), (b, tot)


def test_long_context_prompt_tail():
    """Two 32768-token prompts at the long32k head shape (Hq=40, Hkv=8): the last 48
    tokens of three tables against the oracle (they depend only on the last 48
    queries, each over its whole causal row), every score finite and in (0, 1]."""
    cfg = inputs.CONFIGS["long32k"]
    N, Hq, Hkv = 32768, cfg["Hq"], cfg["Hkv"]
    w = inputs.prefill("long32k", B=2)
    new_len = w["new_len"]
    assert list(new_len) == [N, N]
    rows = 2 * N
    q = inputs.prompt_queries("long32k", rows)
    print("case: prompt significance, two 32768-token prompts (Hq %d, Hkv %d)" % (Hq, Hkv), flush=True)
    got = dk.prompt_significance(LD, t(new_len), t(q).view(torch.float16), t(w["k"]).view(torch.float16), SCALE)
    torch.cuda.synchronize()
    g = got.cpu().numpy()
    assert np.all(np.isfinite(g)) and np.all(g >= 0) and np.all(g <= 1.0 + 1e-6)
    m = 48
    for b, h in ((0, 0), (1, 3), (1, 7)):
        print("case: oracle tail, sequence %d head %d" % (b, h), flush=True)
        r0 = b * N
        want = orc.prompt_significance_tail(q[r0:r0 + N], w["k"][r0:r0 + N], SCALE, h, m)
        _close(g[r0 + N - m:r0 + N, h], want, "32k tail (%d, %d)" % (b, h))
