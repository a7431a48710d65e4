"""Helpers of the GPU parity tests: move cache state between the oracle (numpy) and the
HIP library (torch device tensors), and compare them."""
import numpy as np
import torch

from oracle import oracle as orc
from paper_2412_03131_amd import diffkv as dk

DEV = torch.device("cuda:0")
ATOL = 2e-3   # max |out_gpu - out_oracle|
RTOL = 1e-3   # ||out_gpu - out_oracle||_2 / ||out_oracle||_2


def t(a):
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        a = a.view(np.int16)
    if a.dtype == np.uint32:
        a = a.view(np.int32)
    return torch.from_numpy(a).to(DEV)


def layouts(**kw):
    return orc.layout(**kw), dk.layout(**kw)


def dev_cache_from_oracle(Ld, oc, with_pool=True):
    """Device cache holding exactly the oracle cache's state."""
    dc = dk.Cache(Ld, oc.num_pages, oc.num_seqs, oc.num_kv_heads, device=DEV, with_pool=with_pool)
    if with_pool:
        dc.pool.copy_(t(oc.pool))
    dc.page_table.copy_(t(oc.table))
    dc.pages.copy_(t(oc.pages))
    dc.len.copy_(t(oc.len))
    dc.seq_len.copy_(t(oc.seq_len))
    dc.ring.copy_(t(oc.ring))
    dc.ring_ptr.copy_(t(oc.ring_ptr))
    dc.status.copy_(t(oc.status.view(np.int32)))
    return dc


def snapshot(dc, with_pool=True):
    torch.cuda.synchronize()
    s = dict(table=dc.page_table.cpu().numpy(), pages=dc.pages.cpu().numpy(),
             len=dc.len.cpu().numpy(), seq_len=dc.seq_len.cpu().numpy(),
             ring=dc.ring.cpu().numpy(), ring_ptr=dc.ring_ptr.cpu().numpy(),
             status=dc.status.cpu().numpy().view(np.uint32))
    if with_pool:
        s["pool"] = dc.pool.cpu().numpy()
    return s


def assert_state_equal(dc, oc, with_pool=True, what=""):
    s = snapshot(dc, with_pool)
    for f, o in (("table", oc.table), ("pages", oc.pages), ("len", oc.len),
                 ("seq_len", oc.seq_len), ("ring", oc.ring), ("ring_ptr", oc.ring_ptr),
                 ("status", oc.status)):
        assert np.array_equal(s[f], o), "%s: %s differs" % (what, f)
    if with_pool:
        # every page that holds tokens, byte for byte (fresh pages are zero-filled on both sides)
        used = []
        for tt in range(oc.num_tables):
            for sec in (0, 1):
                T = oc.L.tokens_per_page[sec]
                npg = -(-int(oc.len[tt, sec]) // T)
                for k in range(npg):
                    slot = k if sec == 0 else oc.L.p_max - 1 - k
                    used.append(int(oc.table[tt, slot]))
        used = np.array(sorted(set(used)), np.int64)
        if len(used):
            bad = np.where((s["pool"][used] != oc.pool[used]).any(axis=1))[0]
            assert len(bad) == 0, "%s: %d of %d pages differ, first page %d" % (
                what, len(bad), len(used), used[bad[0]])
    return s


def attention_errors(out, ref):
    out = np.asarray(out, np.float64)
    d = np.abs(out - ref)
    rel = np.linalg.norm(out - ref) / max(np.linalg.norm(ref), 1e-300)
    return float(d.max()), float(rel)


def assert_attention_close(out, lse, ref, ref_lse, what=""):
    mx, rel = attention_errors(out, ref)
    assert mx <= ATOL and rel <= RTOL, "%s: max abs %.3g, rel L2 %.3g" % (what, mx, rel)
    if lse is not None:
        lse = np.asarray(lse, np.float64)
        fin = np.isfinite(ref_lse)
        assert np.array_equal(np.isfinite(lse), fin), what + ": lse finiteness"
        assert np.abs(lse[fin] - ref_lse[fin]).max(initial=0.0) <= 2e-3, what + ": lse"
    return mx, rel
