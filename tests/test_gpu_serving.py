"""GPU parity of the request lifecycle at serving scale (Sec. 5.3: completion recycling;
memory management run once per inference step for all requests and all layers).

The bench's serving step on a reduced llama8b shape: three layers of eight sequences
(32 query / 8 KV heads) share one page pool; "sequence" l*B + b of the cache is
sequence b of layer l.  Each of ten steps

  1. finishes request r = step mod B: one compaction call releases every live slot of
     its tables in every layer (and its sequence lengths are reset);
  2. makes one append call for all layers: request r is prefilled anew with a prompt
     while the other sequences append one decode token (quota (1, 0));
  3. runs attention per layer over that layer's cache view.

After every step the whole state (pool bytes of every used page, tables, page counts,
lengths, sequence lengths, the ring and its pointers, status) must equal the oracle's
bit for bit, and every layer's attention output must be within the tolerance.
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


@pytest.mark.parametrize("splits", [0, -1])
def test_serving_steps_multi_layer(splits):
    B, NL, steps = 8, 3, 10
    w = inputs.prefill("llama8b", B=B, L=(200, 600))
    Hq, Hkv = w["Hq"], w["Hkv"]
    nl = w["new_len"].astype(np.int64)
    off = np.concatenate([[0], np.cumsum(nl)])
    per = (-(-(w["quota"][:, :, 0].astype(np.int64) + steps) // 16)) + (-(-w["quota"][:, :, 1] // 32)) + 2
    npages = int(NL * per.sum() * 1.3) + 64
    Lo, Ld = layouts(max_seq_len=int(nl.max()) + steps + 16)
    oc = orc.Cache(Lo, npages, NL * B, Hkv, ring=np.random.default_rng(51).permutation(npages))
    dc = dev_cache_from_oracle(Ld, oc)
    views = [dc.view(l * B, (l + 1) * B) for l in range(NL)]

    def append(new_len, k, v, score, quota):
        orc.quantize_append(oc, new_len, k, v, score, quota=quota)
        dk.quantize_append(dc, t(new_len.astype(np.int32)), t(k), t(v), t(score),
                           quota=t(quota.astype(np.int32)), total_new=int(new_len.sum()),
                           max_new=int(new_len.max()))

    # prompt phase of every request in every layer, one call
    print("case: serving prompt phase, %d layers x %d sequences" % (NL, B), flush=True)
    append(np.tile(w["new_len"], NL), np.concatenate([w["k"]] * NL), np.concatenate([w["v"]] * NL),
           np.concatenate([w["score"]] * NL), np.tile(w["quota"], (NL, 1, 1)))
    assert oc.status[0] == 0
    assert_state_equal(dc, oc, what="serving prompt")
    P = Lo.p_max
    for s in range(steps):
        r = s % B
        print("case: serving step %d (request %d finishes and is re-prefilled)" % (s, r), flush=True)
        # 1. request r finishes in every layer: one compaction for all layers
        rel = np.zeros((NL * B * Hkv, P), np.uint8)
        for l in range(NL):
            rel[(l * B + r) * Hkv:(l * B + r + 1) * Hkv] = 1
        orc.compact(oc, rel)
        dk.compact_free_list(dc, t(rel))
        oc.seq_len[r::B] = 0
        dc.seq_len[r::B] = 0
        # 2. one append for all layers: request r re-prefilled, the others decode
        d = inputs.decode_token("llama8b", s, B, Hq, Hkv, w["outliers"])
        n_np = np.ones(B, np.int64)
        n_np[r] = nl[r]
        rows_k = [d["k"][:r], w["k"][off[r]:off[r + 1]], d["k"][r + 1:]]
        rows_v = [d["v"][:r], w["v"][off[r]:off[r + 1]], d["v"][r + 1:]]
        rows_s = [d["score"][:r], w["score"][off[r]:off[r + 1]], d["score"][r + 1:]]
        quota = d["quota"].copy()
        quota[r] = w["quota"][r]
        append(np.tile(n_np, NL), np.concatenate(rows_k * NL), np.concatenate(rows_v * NL),
               np.concatenate(rows_s * NL), np.tile(quota, (NL, 1, 1)))
        assert oc.status[0] == 0
        assert_state_equal(dc, oc, what="serving step %d" % s)
        # 3. attention per layer (the oracle computes all layers' sequences at once)
        q_all = np.concatenate([d["q"]] * NL)
        ref, ref_lse = orc.attention(oc, q_all, SCALE)
        for l in range(NL):
            out, lse = dk.decode_attention(views[l], t(d["q"]), SCALE, num_splits=splits)
            torch.cuda.synchronize()
            assert_attention_close(out.cpu().numpy(), lse.cpu().numpy(), ref[l * B:(l + 1) * B],
                                   ref_lse[l * B:(l + 1) * B], "serving step %d layer %d" % (s, l))
    # the ring holds every page exactly once: the free region plus the live table entries
    head, tail = (int(x) for x in oc.ring_ptr)
    free = oc.ring[np.arange(head, tail) % npages]
    live = oc.table[oc.table >= 0]
    assert np.array_equal(np.sort(np.concatenate([free, live])), np.arange(npages))
