"""GPU parity of the generation-phase policy (Sec. 4, Algorithm 1) against the CPU
oracle, state compared bit for bit (page bytes, tables, lengths, ring):

  - every branch of the rule on the one-table worked cases the oracle is pinned on;
  - multi-step runs on ragged tables (one table shorter than the window, victims in
    both sections, swap-removes across pages, low sections growing a page);
  - refusal: a ring too short for the low pages a step needs (OUT_OF_PAGES) and
    tables at their width (TABLE_OVERFLOW) leave the cache unchanged on both sides;
  - the llama8b workload at full size with the 64-token window, then attention.

Decode-token scores are the generator's uniform draws scaled to [0, 2/N), the scale
of the prompt's normalized scores, so every branch of the rule occurs.
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
from test_oracle_generation import ALPHA_H as CASE_AH, ALPHA_L as CASE_AL  # noqa: E402
from test_oracle_generation import W as CASE_W, _prompt_then_decode  # noqa: E402

SCALE = 1.0 / np.sqrt(128.0)


@pytest.mark.parametrize("prompt,cand", [
    ([0.08, 0.09, 0.07, 0.06, 0.01, 0.02], 0.5),     # high victim moves low
    ([0.03, 0.04, 0.02, 0.015, 0.01, 0.005], 0.5),   # high victim removed
    ([0.3, 0.4, 0.2, 0.06, 0.01, 0.02], 0.5),        # high victim stays
    ([0.3, 0.4, 0.2, 0.01, 0.005, 0.002], 0.07),     # candidate low, low victim evicted
    ([0.3, 0.4, 0.2, 0.06, 0.005, 0.002], 0.07),     # candidate low, appended
    ([0.3, 0.4, 0.2, 0.06, 0.005, 0.002], 0.01),     # candidate removed
    ([0.08, 0.08, 0.07, 0.06, 0.01, 0.02], 0.5),     # equal lowest scores: lower position
])
def test_branches_match_oracle(prompt, cand):
    oc = _prompt_then_decode(orc, prompt, cand)
    Ld = dk.layout(max_seq_len=64)
    dc = dev_cache_from_oracle(Ld, oc)
    print("case: generation branch prompt=%s cand=%s" % (prompt, cand), flush=True)
    orc.generation_step(oc, CASE_AH, CASE_AL, CASE_W)
    dk.generation_step(dc, CASE_AH, CASE_AL, CASE_W)
    assert_state_equal(dc, oc, what="branch %s %s" % (prompt, cand))


def _prompt(seed, lens, Hkv, f_hi, f_pr):
    r_k, r_v, r_s, r_o = [np.random.default_rng(s) for s in np.random.SeedSequence(seed).spawn(4)]
    outl = inputs.outlier_channels(r_o, Hkv)
    lens = np.asarray(lens, np.int32)
    k, v = inputs.draw_kv(r_k, r_v, int(lens.sum()), Hkv, outl)
    score = np.empty((int(lens.sum()), Hkv), np.float32)
    quota = np.zeros((len(lens), Hkv, 2), np.int32)
    off = 0
    for b, n in enumerate(lens):
        for h in range(Hkv):
            score[off:off + n, h] = inputs.zipf_scores(r_s, int(n))
        nh, nl = inputs.counts_from_fractions(int(n), np.full(Hkv, f_hi), np.full(Hkv, f_pr))
        quota[b, :, 0], quota[b, :, 1] = nh, nl
        off += n
    return lens, k, v, score, quota, outl


def _append_both(oc, dc, new_len, k, v, score, quota, window):
    orc.quantize_append(oc, new_len, k, v, score, quota=quota, window=window)
    dk.quantize_append(dc, t(np.asarray(new_len, np.int32)), t(k), t(v), t(score),
                       quota=t(np.asarray(quota, np.int32)), window=window,
                       total_new=int(np.sum(new_len)), max_new=int(np.max(new_len, initial=0)))


def _decode(seed, step, B, Hkv, outl, seq_len):
    d = inputs.decode_token("tiny", step, B, 2 * Hkv, Hkv, outl, seed=seed)
    n = (np.asarray(seq_len, np.int64) + 1).astype(np.float32)
    d["score"] = (d["score"] * (np.float32(2.0) / n)[:, None]).astype(np.float32)
    return d


def _clear_status(oc, dc):
    oc.status[0] = 0
    dc.status.zero_()


def _run(seed, lens, Hkv, W, steps, npages, max_seq_len, alpha=(1.0, 0.5), check=None,
         f_hi=0.3, f_pr=0.3, free_after_prompt=None):
    """Prompt append, then `steps` decode steps (append + generation step) on both
    sides; state compared after the steps in `check` (all when None).  The status
    word is cleared before each call, so `seen["refused"]` counts generation steps
    that raised a bit.  `free_after_prompt` shrinks the free region (tail = head + n)
    on both sides after the prompt."""
    lens, k, v, score, quota, outl = _prompt(seed, lens, Hkv, f_hi, f_pr)
    B = len(lens)
    Lo, Ld = layouts(max_seq_len=max_seq_len)
    ring = np.random.default_rng(seed + 1).permutation(npages)
    oc = orc.Cache(Lo, npages, B, Hkv, ring=ring)
    dc = dev_cache_from_oracle(Ld, oc)
    _append_both(oc, dc, lens, k, v, score, quota, W)
    assert int(oc.status[0]) == 0
    if free_after_prompt is not None:
        oc.ring_ptr[1] = oc.ring_ptr[0] + free_after_prompt
        dc.ring_ptr.copy_(t(oc.ring_ptr))
    assert_state_equal(dc, oc, what="prompt")
    seen = dict(low_grew=0, high_only=0, page_taken=0, refused=0, bits=0)
    for step in range(steps):
        d = _decode(seed, step, B, Hkv, outl, oc.seq_len)
        _append_both(oc, dc, d["new_len"], d["k"], d["v"], d["score"], d["quota"], W)
        if check is None or step in check:
            assert_state_equal(dc, oc, what="seed %d append %d" % (seed, step))
        _clear_status(oc, dc)
        before_len, before_pages = oc.len.copy(), oc.pages.copy()
        print("case: seed %d generation step %d" % (seed, step), flush=True)
        orc.generation_step(oc, alpha[0], alpha[1], W)
        dk.generation_step(dc, alpha[0], alpha[1], W)
        if check is None or step in check:
            assert_state_equal(dc, oc, what="seed %d step %d" % (seed, step))
        dl = oc.len - before_len
        seen["low_grew"] += int((dl[:, 1] == 1).sum())
        seen["high_only"] += int(((dl[:, 0] == -1) & (dl[:, 1] == 0)).sum())
        seen["page_taken"] += int((oc.pages - before_pages).sum())
        seen["refused"] += int(int(oc.status[0]) != 0)
        seen["bits"] |= int(oc.status[0])
        if int(oc.status[0]):
            assert np.array_equal(oc.len, before_len) and np.array_equal(oc.pages, before_pages)
        _clear_status(oc, dc)
    return oc, dc, seen


def test_ragged_multi_step():
    """Five sequences (one shorter than the window), two KV heads, 48 steps."""
    oc, dc, seen = _run(11, [3, 40, 77, 130, 200], 2, 8, 48, 400, 512)
    assert seen["refused"] == 0
    assert seen["low_grew"] > 0 and seen["high_only"] > 0 and seen["page_taken"] > 0
    q = inputs.f16_bits(np.random.default_rng(5).standard_normal((5, 4, 128)).astype(np.float32))
    ref, ref_lse = orc.attention(oc, q, SCALE)
    for splits in (1, 0, -1):
        out, lse = dk.decode_attention(dc, t(q), SCALE, num_splits=splits)
        torch.cuda.synchronize()
        assert_attention_close(out.cpu().numpy(), lse.cpu().numpy(), ref, ref_lse,
                               "after generation steps, splits %d" % splits)


def test_window_zero_and_single_head():
    """W = 0: the candidate is the token the step's append just added."""
    oc, dc, seen = _run(12, [17, 33, 64, 90], 1, 0, 24, 200, 256, alpha=(0.8, 0.3))
    assert seen["refused"] == 0 and seen["high_only"] > 0


def test_out_of_pages_refused_identically():
    """A ring with a few spare pages: steps that need low pages are refused
    all-or-nothing (status bit, nothing changed) the same way on both sides."""
    oc, dc, seen = _run(13, [60, 90, 120], 2, 4, 40, 256, 256, alpha=(1.5, 0.2), f_hi=0.6,
                        f_pr=0.1, free_after_prompt=3)
    assert seen["refused"] > 0 and seen["bits"] == dk.ST_OUT_OF_PAGES


def test_table_overflow_refused_identically():
    """Tables at their width: a step whose low section needs one more page is
    refused with TABLE_OVERFLOW on both sides."""
    oc, dc, seen = _run(14, [92, 92], 2, 4, 80, 256, 80, alpha=(1.5, 0.2), f_hi=0.6, f_pr=0.1)
    assert seen["refused"] > 0 and seen["bits"] == dk.ST_TABLE_OVERFLOW


@pytest.mark.parametrize("nseq,free", [(520, None), (520, 40), (200, None)])
def test_many_tables(nseq, free):
    """Many tables: 4160 (520 sequences x 8 KV heads, more than an apply wave plans
    for: the allocation is planned by its own kernel; with a short ring, steps are
    refused) and 1600 (each apply wave plans over two rounds of page requests)."""
    lens = np.random.default_rng(15).integers(6, 60, nseq)
    oc, dc, seen = _run(15, lens, 8, 4, 4, 24000, 128, alpha=(1.5, 0.2), f_hi=0.5,
                        f_pr=0.1, free_after_prompt=free)
    assert oc.num_tables in (4160, 1600) and seen["page_taken"] + seen["refused"] > 0
    if free is None:
        assert seen["refused"] == 0 and seen["page_taken"] > 0
    else:
        assert seen["refused"] > 0 and seen["bits"] == dk.ST_OUT_OF_PAGES


def test_long_context_tables():
    """Two sequences of 12000 and 9000 tokens (high sections of ~4000-8000 tokens):
    every decide thread walks several rounds of 2048-token chunks."""
    oc, dc, seen = _run(16, [12000, 9000], 2, 64, 6, 2400, 12160, alpha=(1.0, 0.5),
                        f_hi=0.6, f_pr=0.1, check={0, 5})
    assert seen["refused"] == 0 and max(oc.len[:, 0]) > 4096


def test_full_size_llama8b_window64():
    """The llama8b workload (B = 64, Hkv = 8, contexts 1024-4096) at full size with the
    64-token window: prompt append, six decode steps with the generation policy,
    then attention in the automatic mode."""
    W = 64
    w = inputs.prefill("llama8b")
    B, Hq, Hkv = w["B"], w["Hq"], w["Hkv"]
    quota = w["quota"]
    per = (-(-quota[:, :, 0] // 16)) + (-(-quota[:, :, 1] // 32)) + 8
    npages = int(per.sum()) + 1024
    Lo, Ld = layouts(max_seq_len=int(w["max_len"]) + 64)
    oc = orc.Cache(Lo, npages, B, Hkv, ring=np.random.default_rng(43).permutation(npages))
    dc = dev_cache_from_oracle(Ld, oc)
    print("case: llama8b full-size prompt append, window 64", flush=True)
    _append_both(oc, dc, w["new_len"], w["k"], w["v"], w["score"], quota, W)
    assert oc.status[0] == 0
    outl = w["outliers"]
    del w
    changed = 0
    for step in range(6):
        d = _decode(1, step, B, Hkv, outl, oc.seq_len)
        d["q"] = inputs.decode_token("llama8b", step, B, Hq, Hkv, outl)["q"]
        _append_both(oc, dc, d["new_len"], d["k"], d["v"], d["score"], d["quota"], W)
        before = oc.len.copy()
        print("case: llama8b full-size generation step %d" % step, flush=True)
        orc.generation_step(oc, 1.0, 0.5, W)
        dk.generation_step(dc, 1.0, 0.5, W)
        changed += int((oc.len != before).any(axis=1).sum())
        if step in (0, 1, 5):
            assert_state_equal(dc, oc, what="llama8b full-size generation step %d" % step)
    assert oc.status[0] == 0 and changed > 0
    ref, ref_lse = orc.attention(oc, d["q"], SCALE)
    out, lse = dk.decode_attention(dc, t(d["q"]), SCALE, num_splits=0)
    torch.cuda.synchronize()
    assert_attention_close(out.cpu().numpy(), lse.cpu().numpy(), ref, ref_lse,
                           "llama8b after generation steps")
