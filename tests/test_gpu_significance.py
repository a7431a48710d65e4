"""GPU parity of the significance update (Sec. 4; diffkv_update_significance) against the
oracle: after diffkv_decode_attention, every kept token's score is rewritten as the
running mean of its attention probability (max over the KV head's query heads).

Every byte of every used page outside the score segments must stay bit-identical to the
oracle's; the scores must agree within 1e-4 relative (fp32 logits and exp2 on the GPU,
fp64 in the oracle).  Cases: every group size 1-8 on high-only, low-only and mixed
tables with ragged tails; empty tables and single tokens; decode steps with appends
between updates; the full llama8b decode workload.
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

from gpu_util import dev_cache_from_oracle, layouts, t  # noqa: E402

SCALE = 1.0 / np.sqrt(128.0)
RTOL = 1e-4   # the newest token's score is its probability: exp(logit - lse) carries the fp32 logit error (up to ~5e-5)


def _score_mask(L):
    """Per page: True on the bytes of the score segments of both precisions."""
    m = np.zeros(L.page_bytes, bool)
    for sec in (0, 1):
        m[L.off_score[sec]:L.off_score[sec] + 4 * L.tokens_per_page[sec]] = True
    return m


def _compare(dc, oc, what):
    torch.cuda.synchronize()
    L = oc.L
    pool = dc.pool.cpu().numpy()
    used = np.unique(oc.table[oc.table >= 0])
    m = _score_mask(L)
    a, b = pool[used], oc.pool[used]
    assert np.array_equal(a[:, ~m], b[:, ~m]), what + ": bytes outside the score segments differ"
    nscored = 0
    for tt in range(oc.num_tables):
        for sec in (0, 1):
            T = L.tokens_per_page[sec]
            n = int(oc.len[tt, sec])
            for k in range(-(-n // T)):
                slot = k if sec == 0 else L.p_max - 1 - k
                pid = int(oc.table[tt, slot])
                cnt = min(T, n - k * T)
                o = L.off_score[sec]
                g = pool[pid, o:o + 4 * cnt].view(np.float32).astype(np.float64)
                r = oc.pool[pid, o:o + 4 * cnt].view(np.float32).astype(np.float64)
                assert np.all(np.abs(g - r) <= RTOL * np.abs(r) + 1e-9), (what, tt, sec, k)
                nscored += cnt
    return nscored


def _step(dc, oc, q, splits=0):
    out, lse = dk.decode_attention(dc, t(q), SCALE, num_splits=splits)
    dk.update_significance(dc, t(q), SCALE, lse)
    orc.update_significance(oc, q, SCALE)


@pytest.mark.parametrize("Hkv,Hq", [(4, 4), (2, 4), (1, 3), (2, 8), (1, 5), (2, 12), (1, 7), (1, 8)])
def test_significance_every_group_size(Hkv, Hq):
    rng = np.random.default_rng(60 + Hq)
    B = 3
    new_len = np.array([16, 75, 230], np.int32)
    n = int(new_len.sum())
    k = (rng.standard_normal((n, Hkv, 128)) * 2).astype(np.float16).view(np.uint16)
    v = rng.standard_normal((n, Hkv, 128)).astype(np.float16).view(np.uint16)
    score = (rng.random((n, Hkv)) * 0.01).astype(np.float32)
    quota = np.zeros((B, Hkv, 2), np.int32)
    quota[0, :] = [16, 0]
    quota[1, :] = [0, 75]
    quota[2, :] = [101, 90]
    Lo, Ld = layouts(max_seq_len=256)
    npages = B * Hkv * 20
    oc = orc.Cache(Lo, npages, B, Hkv, ring=rng.permutation(npages))
    orc.quantize_append(oc, new_len, k, v, score, quota=quota)
    dc = dev_cache_from_oracle(Ld, oc)
    q = rng.standard_normal((B, Hq, 128)).astype(np.float16).view(np.uint16)
    print("case: significance, group size %d" % (Hq // Hkv), flush=True)
    _step(dc, oc, q, splits=1)
    assert _compare(dc, oc, "group size %d" % (Hq // Hkv)) > 0


def test_significance_edge_cases_and_steps():
    """Empty tables, single kept tokens, a lone partial page; then decode steps (one
    appended token, then attention and the update) so that the newest tokens count 1."""
    rng = np.random.default_rng(66)
    B, Hkv, Hq = 4, 2, 8
    new_len = np.array([0, 1, 40, 5], np.int32)
    n = int(new_len.sum())
    k = rng.standard_normal((n, Hkv, 128)).astype(np.float16).view(np.uint16)
    v = rng.standard_normal((n, Hkv, 128)).astype(np.float16).view(np.uint16)
    score = rng.random((n, Hkv)).astype(np.float32)
    quota = np.array([[[0, 0], [0, 0]], [[1, 0], [0, 1]], [[17, 5], [0, 0]], [[0, 3], [2, 2]]], np.int32)
    Lo, Ld = layouts(max_seq_len=64)
    oc = orc.Cache(Lo, 64, B, Hkv, ring=rng.permutation(64))
    orc.quantize_append(oc, new_len, k, v, score, quota=quota)
    dc = dev_cache_from_oracle(Ld, oc)
    for step in range(6):
        q = rng.standard_normal((B, Hq, 128)).astype(np.float16).view(np.uint16)
        print("case: significance edge cases, step %d" % step, flush=True)
        _step(dc, oc, q, splits=[1, 0, -1, 2, 1, 0][step])
        _compare(dc, oc, "edge step %d" % step)
        nl = np.ones(B, np.int32)
        kd = rng.standard_normal((B, Hkv, 128)).astype(np.float16).view(np.uint16)
        vd = rng.standard_normal((B, Hkv, 128)).astype(np.float16).view(np.uint16)
        sd = rng.random((B, Hkv)).astype(np.float32)
        qa = np.tile(np.array([1, 0], np.int32), (B, Hkv, 1))
        orc.quantize_append(oc, nl, kd, vd, sd, quota=qa)
        dk.quantize_append(dc, t(nl), t(kd), t(vd), t(sd), quota=t(qa), total_new=B, max_new=1)


def test_significance_full_llama8b():
    w = inputs.prefill("llama8b")
    B, Hq, Hkv = w["B"], w["Hq"], w["Hkv"]
    quota = w["quota"]
    per = (-(-quota[:, :, 0] // 16)) + (-(-quota[:, :, 1] // 32)) + 2
    npages = int(per.sum()) + 256
    Lo, Ld = layouts(max_seq_len=int(w["max_len"]) + 16)
    oc = orc.Cache(Lo, npages, B, Hkv, ring=np.random.default_rng(67).permutation(npages))
    orc.quantize_append(oc, w["new_len"], w["k"], w["v"], w["score"], quota=quota)
    dc = dev_cache_from_oracle(Ld, oc)
    print("case: significance, full llama8b (B=64, Hq=32, Hkv=8)", flush=True)
    _step(dc, oc, w["q"])
    n = _compare(dc, oc, "full llama8b")
    assert n == int(oc.len.sum())
