"""GPU parity at the full size of the timed workload (llama8b decode: B = 64,
Hq = 32, Hkv = 8, contexts 1024-4096), in the launch configuration the bench
times (automatic split mode), against the CPU oracle on every output.

The oracle handles this size in seconds: the prompt-phase append is compared
byte for byte over every used page, then attention over the whole cache, then
two decode steps (one token per table, partial pages) and attention again.
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


def test_llama8b_full_size_append_and_attention():
    w = inputs.prefill("llama8b")
    B, Hq, Hkv = w["B"], w["Hq"], w["Hkv"]
    assert (B, Hq, Hkv) == (64, 32, 8)
    quota = w["quota"]
    # pages for the prompt plus the decode steps, and some spare
    per = (-(-quota[:, :, 0] // 16)) + (-(-quota[:, :, 1] // 32)) + 2
    npages = int(per.sum()) + 256
    Lo, Ld = layouts(max_seq_len=int(w["max_len"]) + 64)
    oc = orc.Cache(Lo, npages, B, Hkv, ring=np.random.default_rng(41).permutation(npages))
    dc = dev_cache_from_oracle(Ld, oc)
    print("case: full-size prompt append (%d rows)" % int(w["new_len"].sum()), flush=True)
    _append_both(oc, dc, w["new_len"], w["k"], w["v"], w["score"], quota)
    assert oc.status[0] == 0
    assert_state_equal(dc, oc, what="full-size prompt append")
    _attention_both(oc, dc, w["q"], "after the prompt")
    for step in range(2):
        d = inputs.decode_token("llama8b", step, B, Hq, Hkv, w["outliers"])
        print("case: full-size decode append, step %d" % step, flush=True)
        _append_both(oc, dc, d["new_len"], d["k"], d["v"], d["score"], d["quota"])
        assert oc.status[0] == 0
        assert_state_equal(dc, oc, what="full-size decode step %d" % step)
        _attention_both(oc, dc, d["q"], "after decode step %d" % step)
