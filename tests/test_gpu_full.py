"""GPU parity at full workload sizes, in the automatic split mode the bench
times, against the CPU oracle on every output:

  llama8b   B = 64, Hq = 32, Hkv = 8, contexts 1024-4096 (the timed workload;
            one workgroup per table)
  llama70b  B = 32, Hq = 64, Hkv = 8, context 8192 (balanced shares + merge)
  long32k   B = 16, Hq = 40, Hkv = 8, context 32768 (balanced shares + merge)

The oracle handles these sizes in seconds: the prompt-phase append is compared
byte for byte over every used page, then attention over the whole cache, then
decode steps (one token per table, partial pages) and attention again.
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

from gpu_util import (assert_attention_close, assert_state_equal,  # noqa: E402
                      dev_cache_from_oracle, layouts, t)

SCALE = 1.0 / np.sqrt(128.0)


def _append_both(oc, dc, new_len, k, v, score, quota):
    orc.quantize_append(oc, new_len, k, v, score, quota=quota)
    dk.quantize_append(dc, t(np.asarray(new_len, np.int32)), t(k), t(v), t(score),
                       quota=t(np.asarray(quota, np.int32)),
                       total_new=int(np.sum(new_len)), max_new=int(np.max(new_len, initial=0)))


def _attention_both(oc, dc, q, what):
    ref, ref_lse = orc.attention(oc, q, SCALE)
    print("case: full-size attention %s (automatic split mode)" % what, flush=True)
    out, lse = dk.decode_attention(dc, t(q), SCALE, num_splits=0)
    torch.cuda.synchronize()
    mx, rel = assert_attention_close(out.cpu().numpy(), lse.cpu().numpy(), ref, ref_lse,
                                     "full-size " + what)
    print("   max abs %.2e rel %.2e" % (mx, rel), flush=True)


@pytest.mark.parametrize("name,steps,dims", [("llama8b", 2, (64, 32, 8)), ("llama70b", 1, (32, 64, 8)),
                                              ("long32k", 1, (16, 40, 8))])
def test_full_size_append_and_attention(name, steps, dims):
    w = inputs.prefill(name)
    B, Hq, Hkv = w["B"], w["Hq"], w["Hkv"]
    assert (B, Hq, Hkv) == dims
    quota = w["quota"]
    # pages for the prompt plus the decode steps, and some spare
    per = (-(-quota[:, :, 0] // 16)) + (-(-quota[:, :, 1] // 32)) + 2
    npages = int(per.sum()) + 256
    Lo, Ld = layouts(max_seq_len=int(w["max_len"]) + 64)
    oc = orc.Cache(Lo, npages, B, Hkv, ring=np.random.default_rng(41).permutation(npages))
    dc = dev_cache_from_oracle(Ld, oc)
    print("case: %s full-size prompt append (%d rows)" % (name, int(w["new_len"].sum())), flush=True)
    _append_both(oc, dc, w["new_len"], w["k"], w["v"], w["score"], quota)
    assert oc.status[0] == 0
    assert_state_equal(dc, oc, what="%s full-size prompt append" % name)
    q, outl = w["q"], w["outliers"]
    del w
    _attention_both(oc, dc, q, "%s after the prompt" % name)
    for step in range(steps):
        d = inputs.decode_token(name, step, B, Hq, Hkv, outl)
        print("case: %s full-size decode append, step %d" % (name, step), flush=True)
        _append_both(oc, dc, d["new_len"], d["k"], d["v"], d["score"], d["quota"])
        assert oc.status[0] == 0
        assert_state_equal(dc, oc, what="%s full-size decode step %d" % (name, step))
        _attention_both(oc, dc, d["q"], "%s after decode step %d" % (name, step))


def test_full_size_compaction_rounds():
    """The compaction workload at full size: 2^20 pages, 4096 tables of up to 256
    slots, 60 % held, Bernoulli(0.35) releases and refill per round; six rounds,
    so the ring wraps.  Every table, length, ring entry and pointer bit-exact."""
    ring, demand = inputs.compaction_setup()
    assert ring.size == 1 << 20 and demand.shape == (4096, 2)
    Lo, Ld = layouts(max_seq_len=255 * 16)
    assert Lo.p_max == 256
    oc = orc.Cache(Lo, 1 << 20, 4096, 1, ring=ring, with_pool=False)
    dc = dev_cache_from_oracle(Ld, oc, with_pool=False)
    orc.alloc_pages(oc, demand)
    dk.alloc_pages(dc, t(demand))
    oc.len[:] = oc.pages * np.array([16, 32])
    dc.len.copy_(t(oc.len))
    assert_state_equal(dc, oc, with_pool=False, what="full-size setup")
    for rnd in range(6):
        print("case: full-size compaction round %d" % rnd, flush=True)
        rel = inputs.release_mask(4, rnd, 4096, 256)
        before = oc.pages.copy()
        orc.compact(oc, rel)
        dk.compact_free_list(dc, t(rel))
        lost = (before - oc.pages).astype(np.int32)
        orc.alloc_pages(oc, lost)
        dk.alloc_pages(dc, t(lost))
        oc.len[:] = oc.pages * np.array([16, 32])
        dc.len.copy_(t(oc.len))
        assert_state_equal(dc, oc, with_pool=False, what="full-size round %d" % rnd)
    assert oc.ring_ptr[1] > (1 << 20)  # wrapped
