"""diffkv_decode_attention_noalloc against diffkv_decode_attention, through the C ABI.

The no-allocation entry point runs the same kernels with the library's fixed
per-device scratch instead of a caller workspace, so its outputs must equal the
workspace entry point's bit for bit.  Two calls in a row on one device share the
scratch: the second, on a smaller cache, must not see anything of the first.  A
call whose resolved mode needs more scratch than the fixed array is refused with
DIFFKV_E_SCRATCH and enqueues nothing.
"""
import ctypes as C

import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():  # pragma: no cover
    pytest.skip("needs a GPU", allow_module_level=True)

from oracle import oracle as orc  # noqa: E402
from paper_2412_03131_amd import diffkv as dk  # noqa: E402
from paper_2412_03131_amd import inputs  # noqa: E402

from gpu_util import DEV, dev_cache_from_oracle, layouts, t  # noqa: E402

SCALE = 1.0 / np.sqrt(128.0)


def _cache(B, L, seed):
    w = inputs.prefill("llama8b", B=B, L=L)
    Lo, Ld = layouts(max_seq_len=int(w["max_len"]) + 64)
    npages = int(w["B"] * w["Hkv"] * (int(w["max_len"]) // 16 + 4))
    oc = orc.Cache(Lo, npages, w["B"], w["Hkv"], ring=np.random.default_rng(seed).permutation(npages))
    orc.quantize_append(oc, w["new_len"], w["k"], w["v"], w["score"], quota=w["quota"])
    assert oc.status[0] == 0
    return dev_cache_from_oracle(Ld, oc), t(w["q"])


def _both(dc, q, splits):
    """(workspace entry point, no-allocation entry point) outputs, each through the C ABI."""
    lib = dk.lib()
    B, Hq, D = q.shape
    stream = C.c_void_p(torch.cuda.current_stream().cuda_stream)
    o1 = torch.full((B, Hq, D), 7.0, dtype=torch.float32, device=DEV)
    l1 = torch.full((B, Hq), 7.0, dtype=torch.float32, device=DEV)
    o2, l2 = o1.clone(), l1.clone()
    need = dk.workspace_size(dk.OP_ATTENTION, dc.L, dc.num_seqs, Hq, dc.num_kv_heads, 0, splits)
    ws = torch.empty(max(need, 256), dtype=torch.uint8, device=DEV)
    st = dc.struct()
    rc = lib.diffkv_decode_attention(C.byref(dc.L), C.byref(st), Hq, C.c_void_p(q.data_ptr()), SCALE,
                                     C.c_void_p(o1.data_ptr()), C.c_void_p(l1.data_ptr()), splits,
                                     C.c_void_p(ws.data_ptr()), ws.numel(), stream)
    assert rc == dk.OK
    rc = lib.diffkv_decode_attention_noalloc(C.byref(dc.L), C.byref(st), Hq, C.c_void_p(q.data_ptr()),
                                             SCALE, C.c_void_p(o2.data_ptr()), C.c_void_p(l2.data_ptr()),
                                             splits, stream)
    assert rc == dk.OK, dk.status_str(rc)
    torch.cuda.synchronize()
    return (o1, l1), (o2, l2)


@pytest.mark.parametrize("splits", [-1, 0, 1, 3])
def test_noalloc_matches_workspace_entry_point(splits):
    big = _cache(6, (300, 1100), 31)
    small = _cache(2, (40, 200), 32)
    for what, (dc, q) in (("first call, 6 sequences", big), ("second call, 2 sequences", small)):
        print("case: no-alloc attention, splits=%d, %s" % (splits, what), flush=True)
        (o1, l1), (o2, l2) = _both(dc, q, splits)
        assert torch.equal(o1, o2), what
        assert torch.equal(l1, l2), what
        assert np.isfinite(o2.cpu().numpy()).all()


def test_noalloc_paired_mode():
    """The automatic mode with at least as many tables as the device holds eight-wave
    workgroups (two per CU) pairs the tables in sixteen-wave workgroups; its only
    scratch is the arrival words.  Two such calls in a row, the second on fewer and
    shorter tables."""
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    b_min = -(-2 * cus // 8) + 1   # llama8b: eight KV heads per sequence
    big = _cache(b_min + 20, (20, 300), 33)
    small = _cache(b_min, (1, 60), 34)
    for what, (dc, q) in (("first call, %d tables" % (8 * (b_min + 20)), big),
                          ("second call, %d tables" % (8 * b_min), small)):
        print("case: no-alloc attention, paired mode, %s" % what, flush=True)
        (o1, l1), (o2, l2) = _both(dc, q, 0)
        assert torch.equal(o1, o2), what
        assert torch.equal(l1, l2), what
        assert np.isfinite(o2.cpu().numpy()).all()


def test_noalloc_refuses_calls_beyond_its_scratch():
    """Balanced shares over 2000 tables of GQ 8: (resident workgroups + 2000) x 8 heads x
    520 B of partial states is more than the 8 MiB scratch; the call is refused and the
    outputs stay untouched.  The automatic mode (one workgroup per table, no partial
    states) fits."""
    Lo, Ld = layouts(max_seq_len=64)
    dc = dk.Cache(Ld, 64, 2000, 1, device=DEV)
    q = torch.zeros((2000, 8, 128), dtype=torch.float16, device=DEV)
    out = torch.full((2000, 8, 128), 7.0, dtype=torch.float32, device=DEV)
    print("case: no-alloc attention beyond the scratch", flush=True)
    with pytest.raises(dk.DiffKVError) as e:
        dk.decode_attention_noalloc(dc, q, SCALE, out, num_splits=-1)
    assert e.value.code == dk.E_SCRATCH
    torch.cuda.synchronize()
    assert bool((out == 7.0).all())
    dk.decode_attention_noalloc(dc, q, SCALE, out, num_splits=0)
    torch.cuda.synchronize()
    assert bool((out == 0.0).all())   # every table is empty: output 0
