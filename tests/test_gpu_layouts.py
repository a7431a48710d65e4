"""GPU parity of the additional precision levels (Sec. 4, Sec. 7.2: K8V8, K8V4, K8V2,
K4V2, K4V1; and 16 tokens per low-precision page): the page layouts the kernels
implement besides K8V4 / K4V2 at 16 / 32 tokens.

For each layout: a prompt-phase append with quotas over ragged sequences and decode
steps of one token into either section, bit-exact against the oracle (every pool byte
of every used page, tables, lengths, ring, pointers); attention in the split modes
1, 3, automatic and balanced for group sizes 1, 4, 5 and 8 within the attention
tolerance; the significance update.  Layouts outside the list are refused.
"""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():  # pragma: no cover
    pytest.skip("needs a GPU", allow_module_level=True)

from oracle import oracle as orc  # noqa: E402
from paper_2412_03131_amd import diffkv as dk  # noqa: E402

from gpu_util import (assert_attention_close, assert_state_equal,  # noqa: E402
                      dev_cache_from_oracle, layouts, t)

SCALE = 1.0 / np.sqrt(128.0)

LAYOUTS = {
    "K8V8-K4V2": dict(k_bits=(8, 4), v_bits=(8, 2), tokens_per_page=(16, 32)),
    "K8V2-K4V1": dict(k_bits=(8, 4), v_bits=(2, 1), tokens_per_page=(16, 32)),
    "K8V4-K4V2-T16": dict(k_bits=(8, 4), v_bits=(4, 2), tokens_per_page=(16, 16)),
}


def _prompt(rng, B, Hkv, new_len):
    n = int(new_len.sum())
    k = (rng.standard_normal((n, Hkv, 128)) * 2).astype(np.float16).view(np.uint16)
    v = rng.standard_normal((n, Hkv, 128)).astype(np.float16).view(np.uint16)
    score = rng.random((n, Hkv)).astype(np.float32)
    quota = np.stack([(new_len[:, None] * rng.uniform(0.1, 0.6, (B, Hkv))).astype(np.int32),
                      (new_len[:, None] * rng.uniform(0.1, 0.5, (B, Hkv))).astype(np.int32)], axis=2)
    return k, v, score, quota


def _append_both(oc, dc, new_len, k, v, score, quota):
    orc.quantize_append(oc, new_len, k, v, score, quota=quota)
    dk.quantize_append(dc, t(new_len.astype(np.int32)), t(k), t(v), t(score), quota=t(quota.astype(np.int32)),
                       total_new=int(new_len.sum()), max_new=int(new_len.max()))


@pytest.mark.parametrize("name", list(LAYOUTS))
def test_layout_append_attention_significance(name):
    kw = LAYOUTS[name]
    rng = np.random.default_rng(100 + len(name))
    B, Hkv = 4, 2
    new_len = np.array([33, 250, 7, 600], np.int32)
    Lo, Ld = layouts(max_seq_len=700, **kw)
    npages = 200
    oc = orc.Cache(Lo, npages, B, Hkv, ring=rng.permutation(npages))
    oc.pool[:] = rng.integers(0, 256, oc.pool.shape, dtype=np.uint8)   # fresh pages must be cleared
    dc = dev_cache_from_oracle(Ld, oc)
    print("case: layout %s, prompt append" % name, flush=True)
    k, v, score, quota = _prompt(rng, B, Hkv, new_len)
    _append_both(oc, dc, new_len, k, v, score, quota)
    assert oc.status[0] == 0
    assert_state_equal(dc, oc, what="%s prompt" % name)
    for step in range(20):
        nl = (rng.random(B) < 0.9).astype(np.int32)
        m = int(nl.sum())
        kd = rng.standard_normal((m, Hkv, 128)).astype(np.float16).view(np.uint16)
        vd = rng.standard_normal((m, Hkv, 128)).astype(np.float16).view(np.uint16)
        sd = rng.random((m, Hkv)).astype(np.float32)
        qa = np.where(rng.random((B, Hkv, 1)) < 0.5, [[1, 0]], [[0, 1]]).astype(np.int32)
        _append_both(oc, dc, nl, kd, vd, sd, qa)
    assert oc.status[0] == 0
    print("case: layout %s, after 20 decode appends" % name, flush=True)
    assert_state_equal(dc, oc, what="%s decode" % name)
    for gq in (1, 4, 5, 8):
        Hq = Hkv * gq
        q = rng.standard_normal((B, Hq, 128)).astype(np.float16).view(np.uint16)
        ref, ref_lse = orc.attention(oc, q, SCALE)
        for splits in (1, 3, 0, -1):
            print("case: layout %s attention GQ %d splits=%d" % (name, gq, splits), flush=True)
            out, lse = dk.decode_attention(dc, t(q), SCALE, num_splits=splits)
            torch.cuda.synchronize()
            mx, rel = assert_attention_close(out.cpu().numpy(), lse.cpu().numpy(), ref, ref_lse,
                                             "%s GQ %d splits %d" % (name, gq, splits))
    # the significance update, after attention with the same q (GQ 4)
    q = rng.standard_normal((B, Hkv * 4, 128)).astype(np.float16).view(np.uint16)
    out, lse = dk.decode_attention(dc, t(q), SCALE)
    dk.update_significance(dc, t(q), SCALE, lse)
    orc.update_significance(oc, q, SCALE)
    torch.cuda.synchronize()
    pool = dc.pool.cpu().numpy()
    for tt in range(B * Hkv):
        for sec in (0, 1):
            T = Lo.tokens_per_page[sec]
            n = int(oc.len[tt, sec])
            for kk in range(-(-n // T)):
                pid = int(oc.table[tt, kk if sec == 0 else Lo.p_max - 1 - kk])
                cnt = min(T, n - kk * T)
                o = Lo.off_score[sec]
                g = pool[pid, o:o + 4 * cnt].view(np.float32).astype(np.float64)
                r = oc.pool[pid, o:o + 4 * cnt].view(np.float32).astype(np.float64)
                assert np.all(np.abs(g - r) <= 1e-4 * np.abs(r) + 1e-9), (name, tt, sec, kk)
    # the generation-phase policy implements K8V4 / K4V2 at 16 / 32 tokens only
    with pytest.raises(dk.DiffKVError) as e:
        dk.generation_step(dc, 1.0, 0.5, 0)
    assert e.value.code == dk.E_UNSUPPORTED


@pytest.mark.parametrize("name", ["K8V4-K4V2"] + list(LAYOUTS))
def test_layout_append_planned(name):
    """Every layout on the path for more than 1024 tables (the plan in a launch of its
    own, then page jobs of fewer waves each): two long prompts among short ones, then
    decode steps into either section, bit-exact against the oracle."""
    kw = LAYOUTS.get(name, dict(k_bits=(8, 4), v_bits=(4, 2), tokens_per_page=(16, 32)))
    rng = np.random.default_rng(300 + len(name))
    B, Hkv = 130, 8
    new_len = rng.integers(0, 30, B).astype(np.int32)
    new_len[[5, 77]] = [700, 333]
    Lo, Ld = layouts(max_seq_len=760, **kw)
    npages = 6000
    oc = orc.Cache(Lo, npages, B, Hkv, ring=rng.permutation(npages))
    oc.pool[:] = rng.integers(0, 256, oc.pool.shape, dtype=np.uint8)
    dc = dev_cache_from_oracle(Ld, oc)
    print("case: layout %s, planned prompt append, %d tables" % (name, B * Hkv), flush=True)
    k, v, score, quota = _prompt(rng, B, Hkv, new_len)
    _append_both(oc, dc, new_len, k, v, score, quota)
    assert oc.status[0] == 0
    assert_state_equal(dc, oc, what="%s planned prompt" % name)
    for step in range(3):
        nl = (rng.random(B) < 0.9).astype(np.int32)
        m = int(nl.sum())
        kd = rng.standard_normal((m, Hkv, 128)).astype(np.float16).view(np.uint16)
        vd = rng.standard_normal((m, Hkv, 128)).astype(np.float16).view(np.uint16)
        sd = rng.random((m, Hkv)).astype(np.float32)
        qa = np.where(rng.random((B, Hkv, 1)) < 0.5, [[1, 0]], [[0, 1]]).astype(np.int32)
        print("case: layout %s, planned decode step %d" % (name, step), flush=True)
        _append_both(oc, dc, nl, kd, vd, sd, qa)
        assert oc.status[0] == 0
        assert_state_equal(dc, oc, what="%s planned step %d" % (name, step))


def test_unsupported_layouts_are_refused():
    for kw in (dict(k_bits=(8, 8), v_bits=(8, 8), tokens_per_page=(16, 16)),
               dict(k_bits=(4, 4), v_bits=(4, 2), tokens_per_page=(16, 32)),
               dict(k_bits=(8, 4), v_bits=(4, 2), tokens_per_page=(16, 64))):
        Ld = dk.layout(max_seq_len=64, **kw)
        dc = dk.Cache(Ld, 8, 1, 1, device="cuda:0")
        q = torch.zeros((1, 1, 128), dtype=torch.float16, device="cuda:0")
        with pytest.raises(dk.DiffKVError) as e:
            dk.decode_attention(dc, q, SCALE)
        assert e.value.code == dk.E_UNSUPPORTED
        one = torch.ones(1, dtype=torch.int32, device="cuda:0")
        kv = torch.zeros((1, 1, 128), dtype=torch.float16, device="cuda:0")
        sc = torch.zeros((1, 1), dtype=torch.float32, device="cuda:0")
        with pytest.raises(dk.DiffKVError) as e:
            dk.quantize_append(dc, one, kv, kv, sc, quota=torch.tensor([[[1, 0]]], dtype=torch.int32,
                                                                       device="cuda:0"), total_new=1, max_new=1)
        assert e.value.code == dk.E_UNSUPPORTED
