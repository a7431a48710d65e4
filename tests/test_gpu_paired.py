"""GPU parity of the automatic attention mode when the tables alone fill the device:
up to GQ 5 each sixteen-wave workgroup takes two tables (ranks j and T-1-j by
decreasing work) and splits its waves between them in proportion to their work.

That path runs only with at least as many tables as the device holds eight-wave
workgroups at once (two per CU), so these caches have 2 * CUs tables or more, most
of them short: empty tables, single tokens, ragged tails, a few long tables paired
with short ones, an odd table count (a workgroup with one table), more tables than
the ranking wave ranks (identity order), every group size 1-5 and every page layout.
Every output is compared with the oracle (max-abs 2e-3, relative L2 1e-3, lse 2e-3),
as are the one-workgroup-per-table (num_splits = 1) results on the same caches.
"""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():  # pragma: no cover
    pytest.skip("needs a GPU", allow_module_level=True)

from oracle import oracle as orc  # noqa: E402
from paper_2412_03131_amd import diffkv as dk  # noqa: E402

from gpu_util import assert_attention_close, dev_cache_from_oracle, layouts, t  # noqa: E402

SCALE = 1.0 / np.sqrt(128.0)
LAYOUTS = {
    "K8V4|K4V2": dict(),
    "K8V8|K4V2": dict(k_bits=(8, 4), v_bits=(8, 2), tokens_per_page=(16, 32)),
    "K8V2|K4V1": dict(k_bits=(8, 4), v_bits=(2, 1), tokens_per_page=(16, 32)),
    "K8V4|K4V2 16/16": dict(k_bits=(8, 4), v_bits=(4, 2), tokens_per_page=(16, 16)),
}


def _min_tables():
    return 2 * torch.cuda.get_device_properties(0).multi_processor_count


def _cache(B, Hkv, new_len, seed, **kw):
    rng = np.random.default_rng(seed)
    n = int(new_len.sum())
    k = (rng.standard_normal((n, Hkv, 128)) * rng.uniform(0.5, 2.0)).astype(np.float16).view(np.uint16)
    v = rng.standard_normal((n, Hkv, 128)).astype(np.float16).view(np.uint16)
    score = rng.random((n, Hkv)).astype(np.float32)
    quota = np.stack([(new_len[:, None] * rng.uniform(0, 0.7, (B, Hkv))).astype(np.int32),
                      (new_len[:, None] * rng.uniform(0, 0.6, (B, Hkv))).astype(np.int32)], axis=2)
    Lo, Ld = layouts(max_seq_len=int(new_len.max(initial=0)) + 64, **kw)
    hi_t, lo_t = Lo.tokens_per_page
    npages = int(sum(-(-int(q[0]) // hi_t) + -(-int(q[1]) // lo_t) for q in quota.reshape(-1, 2))) + 64
    oc = orc.Cache(Lo, npages, B, Hkv, ring=rng.permutation(npages))
    orc.quantize_append(oc, new_len, k, v, score, quota=quota)
    return oc, dev_cache_from_oracle(Ld, oc), rng


def _check(oc, dc, rng, Hq, what):
    q = (rng.standard_normal((oc.num_seqs, Hq, 128)) * rng.uniform(0.5, 2.0)).astype(np.float16).view(np.uint16)
    ref, ref_lse = orc.attention(oc, q, SCALE)
    for splits in (0, 1):
        print("case: %s, splits %d" % (what, splits), flush=True)
        out, lse = dk.decode_attention(dc, t(q), SCALE, num_splits=splits)
        torch.cuda.synchronize()
        assert_attention_close(out.cpu().numpy(), lse.cpu().numpy(), ref, ref_lse, "%s splits %d" % (what, splits))


@pytest.mark.parametrize("gq", [1, 2, 3, 4, 5])
def test_paired_every_group_size(gq):
    """601 tables (odd: the middle workgroup has one table), lengths 0-150 with
    a few empty tables and single tokens, and four long tables (3000-6000 tokens)
    that the pairing puts with the shortest ones."""
    Hkv = 1
    B = max(601, _min_tables() + 1) | 1
    rng = np.random.default_rng(300 + gq)
    new_len = rng.integers(0, 151, B).astype(np.int32)
    new_len[rng.choice(B, 20, replace=False)] = 0
    new_len[rng.choice(B, 20, replace=False)] = 1
    new_len[rng.choice(B, 4, replace=False)] = rng.integers(3000, 6001, 4)
    oc, dc, rng = _cache(B, Hkv, new_len, 310 + gq)
    _check(oc, dc, rng, gq * Hkv, "paired, group size %d, %d tables" % (gq, B * Hkv))


@pytest.mark.parametrize("name", list(LAYOUTS))
def test_paired_every_layout(name):
    """Every page layout at group size 4 (two KV heads per sequence)."""
    Hkv, gq = 2, 4
    B = max(300, _min_tables() // Hkv + 1)
    rng = np.random.default_rng(320)
    new_len = rng.integers(0, 200, B).astype(np.int32)
    new_len[:3] = [4000, 0, 1]
    oc, dc, rng = _cache(B, Hkv, new_len, 321, **LAYOUTS[name])
    _check(oc, dc, rng, gq * Hkv, "paired, layout %s, %d tables" % (name, B * Hkv))


def test_paired_identity_order_and_empty():
    """More tables than the ranking wave ranks (1101 > 64 * 16: pairs by index),
    then a cache of 2 * CUs tables that are all empty."""
    B, Hkv = max(1101, _min_tables() + 1), 1
    rng = np.random.default_rng(330)
    new_len = rng.integers(0, 80, B).astype(np.int32)
    oc, dc, rng = _cache(B, Hkv, new_len, 331)
    _check(oc, dc, rng, 3, "paired, identity order, %d tables" % B)
    B = _min_tables()
    oc, dc, rng = _cache(B, Hkv, np.zeros(B, np.int32), 332)
    _check(oc, dc, rng, 2, "paired, all %d tables empty" % B)
