"""ctypes front end of the CPU oracle (test infrastructure only).

Only tests/, the smoke check and the benchmark's CPU-baseline leg may import
this module.  It marshals numpy arrays into oracle/liboracle_diffkv.so and
adds no arithmetic of its own.
"""
import ctypes as C
import os

import numpy as np

from . import build as _build

_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_build.LIB):
            _build.build()
        _lib = C.CDLL(_build.LIB)
        _setup(_lib)
    return _lib


class Layout(C.Structure):
    _fields_ = [
        ("head_dim", C.c_int32), ("group", C.c_int32),
        ("k_bits", C.c_int32 * 2), ("v_bits", C.c_int32 * 2),
        ("tokens_per_page", C.c_int32 * 2),
        ("max_seq_len", C.c_int32), ("p_max", C.c_int32),
        ("page_bytes", C.c_int64),
        ("off_kcode", C.c_int32 * 2), ("off_kmeta", C.c_int32 * 2),
        ("off_vcode", C.c_int32 * 2), ("off_vmeta", C.c_int32 * 2),
        ("off_score", C.c_int32 * 2), ("off_pos", C.c_int32 * 2),
        ("used_bytes", C.c_int32 * 2),
    ]


class _Cache(C.Structure):
    _fields_ = [
        ("pool", C.c_void_p), ("num_pages", C.c_int64),
        ("table", C.c_void_p), ("pages", C.c_void_p), ("len", C.c_void_p),
        ("seq_len", C.c_void_p), ("ring", C.c_void_p), ("ring_ptr", C.c_void_p),
        ("status", C.c_void_p), ("num_seqs", C.c_int32), ("num_kv_heads", C.c_int32),
    ]


def _p(a):
    return None if a is None else a.ctypes.data_as(C.c_void_p)


def _setup(L):
    vp, i32, i64, f32, f64 = C.c_void_p, C.c_int32, C.c_int64, C.c_float, C.c_double
    L.dko_half_to_float_n.argtypes = [i64, vp, vp]
    L.dko_float_to_half_n.argtypes = [i64, vp, vp]
    L.dko_quantize_group.argtypes = [vp, C.c_int, C.c_int, vp, vp, vp]
    L.dko_layout_init.argtypes = [C.POINTER(Layout), C.c_int, C.c_int, vp, vp, vp, C.c_int]
    L.dko_classify.argtypes = [C.c_int, vp, vp, f32, f32, C.c_int, C.c_int, vp]
    L.dko_alloc_pages.argtypes = [C.POINTER(Layout), C.POINTER(_Cache), C.c_int, vp]
    L.dko_quantize_append.argtypes = [C.POINTER(Layout), C.POINTER(_Cache), vp, vp, vp, vp,
                                      vp, f32, f32, C.c_int]
    L.dko_compact.argtypes = [C.POINTER(Layout), C.POINTER(_Cache), C.c_int, vp]
    L.dko_generation_step.argtypes = [C.POINTER(Layout), C.POINTER(_Cache), f32, f32, C.c_int]
    L.dko_read_token.argtypes = [C.POINTER(Layout), C.POINTER(_Cache), C.c_int, C.c_int,
                                 C.c_int, vp, vp, vp, vp]
    L.dko_attention.argtypes = [C.POINTER(Layout), C.POINTER(_Cache), C.c_int, vp, f64, vp, vp]
    L.dko_attention_partial.argtypes = [C.POINTER(Layout), C.POINTER(_Cache), C.c_int, vp, f64,
                                        C.c_int, C.c_int, C.c_int, C.c_int, vp, vp, vp]
    L.dko_merge_partials.argtypes = [C.c_int, C.c_int, vp, vp, vp, vp, vp]
    L.dko_kv_bits_fraction.argtypes = [C.POINTER(Layout), C.c_int, C.c_int, C.c_int, vp, vp]
    L.dko_update_significance.argtypes = [C.POINTER(Layout), C.POINTER(_Cache), C.c_int, vp, f64]
    L.dko_update_significance.restype = C.c_int
    L.dko_prompt_significance.argtypes = [C.c_int, vp, C.c_int, C.c_int, C.c_int, vp, vp, f64, vp, vp]
    L.dko_prompt_significance.restype = C.c_int
    L.dko_prompt_significance_tail.argtypes = [C.c_int, C.c_int, C.c_int, C.c_int, vp, vp, f64, C.c_int, C.c_int, vp]
    L.dko_prompt_significance_tail.restype = C.c_int
    L.dko_float_to_half.restype = C.c_uint16
    L.dko_float_to_half.argtypes = [f32]
    L.dko_half_to_float.restype = f32
    L.dko_half_to_float.argtypes = [C.c_uint16]
    for name in ("dko_layout_init", "dko_alloc_pages", "dko_quantize_append", "dko_compact",
                 "dko_generation_step", "dko_attention"):
        getattr(L, name).restype = C.c_int
    _ = (i32,)


# ---------------------------------------------------------------- fp16 --
def half_to_float(h):
    h = np.ascontiguousarray(h, dtype=np.uint16)
    out = np.empty(h.shape, np.float32)
    lib().dko_half_to_float_n(h.size, _p(h), _p(out))
    return out


def float_to_half(f):
    f = np.ascontiguousarray(f, dtype=np.float32)
    out = np.empty(f.shape, np.uint16)
    lib().dko_float_to_half_n(f.size, _p(f), _p(out))
    return out


def quantize_group(x_bits, bits):
    """x_bits: fp16 bit patterns (uint16[n]).  Returns (scale16, zero16, codes)."""
    x = np.ascontiguousarray(x_bits, dtype=np.uint16)
    s = np.zeros(1, np.uint16)
    z = np.zeros(1, np.uint16)
    codes = np.zeros(x.size, np.uint8)
    lib().dko_quantize_group(_p(x), x.size, bits, _p(s), _p(z), _p(codes))
    return int(s[0]), int(z[0]), codes


# -------------------------------------------------------------- layout --
def layout(head_dim=128, group=32, k_bits=(8, 4), v_bits=(4, 2),
           tokens_per_page=(16, 32), max_seq_len=4096):
    L = Layout()
    kb = np.array(k_bits, np.int32)
    vb = np.array(v_bits, np.int32)
    tp = np.array(tokens_per_page, np.int32)
    rc = lib().dko_layout_init(C.byref(L), head_dim, group, _p(kb), _p(vb), _p(tp), max_seq_len)
    if rc != 0:
        raise ValueError("oracle: parameters do not describe a layout")
    return L


# --------------------------------------------------------------- cache --
class Cache:
    """Host copy of the whole cache state, as numpy arrays."""

    def __init__(self, L, num_pages, num_seqs, num_kv_heads, ring=None, with_pool=True):
        self.L = L
        self.num_pages = int(num_pages)
        self.num_seqs = int(num_seqs)
        self.num_kv_heads = int(num_kv_heads)
        T = self.num_seqs * self.num_kv_heads
        self.pool = (np.zeros((self.num_pages, L.page_bytes), np.uint8) if with_pool
                     else np.zeros((1, L.page_bytes), np.uint8))
        self.table = np.full((T, L.p_max), -1, np.int32)
        self.pages = np.zeros((T, 2), np.int32)
        self.len = np.zeros((T, 2), np.int32)
        self.seq_len = np.zeros(self.num_seqs, np.int32)
        self.ring = (np.arange(self.num_pages, dtype=np.int32) if ring is None
                     else np.ascontiguousarray(ring, np.int32).copy())
        self.ring_ptr = np.array([0, self.num_pages], np.int64)
        self.status = np.zeros(1, np.uint32)

    @property
    def num_tables(self):
        return self.num_seqs * self.num_kv_heads

    def struct(self):
        return _Cache(_p(self.pool), self.num_pages, _p(self.table), _p(self.pages),
                      _p(self.len), _p(self.seq_len), _p(self.ring), _p(self.ring_ptr),
                      _p(self.status), self.num_seqs, self.num_kv_heads)

    def copy(self):
        c = Cache.__new__(Cache)
        c.__dict__.update({k: (v.copy() if isinstance(v, np.ndarray) else v)
                           for k, v in self.__dict__.items()})
        return c


def classify(score, quota=None, alpha_h=0.0, alpha_l=0.0, seq_len_after=1, window=0):
    s = np.ascontiguousarray(score, np.float32)
    q = None if quota is None else np.ascontiguousarray(quota, np.int32)
    cls = np.zeros(s.size, np.int8)
    lib().dko_classify(s.size, _p(s), _p(q), alpha_h, alpha_l, seq_len_after, window, _p(cls))
    return cls


def alloc_pages(cache, demand):
    d = np.ascontiguousarray(demand, np.int32).reshape(-1, 2)
    st = cache.struct()
    rc = lib().dko_alloc_pages(C.byref(cache.L), C.byref(st), d.shape[0], _p(d))
    if rc != 0:
        raise ValueError("oracle: negative demand")


def quantize_append(cache, new_len, k, v, score, quota=None, alpha_h=0.0, alpha_l=0.0,
                    window=0):
    """k, v: fp16 bit patterns (uint16) [rows][Hkv][D]; score fp32 [rows][Hkv]."""
    nl = np.ascontiguousarray(new_len, np.int32)
    k = np.ascontiguousarray(k, np.uint16)
    v = np.ascontiguousarray(v, np.uint16)
    sc = np.ascontiguousarray(score, np.float32)
    q = None if quota is None else np.ascontiguousarray(quota, np.int32)
    st = cache.struct()
    lib().dko_quantize_append(C.byref(cache.L), C.byref(st), _p(nl), _p(k), _p(v), _p(sc), _p(q),
                              alpha_h, alpha_l, window)


def compact(cache, release):
    r = np.ascontiguousarray(release, np.uint8)
    assert r.shape == (cache.num_tables, cache.L.p_max)
    st = cache.struct()
    lib().dko_compact(C.byref(cache.L), C.byref(st), cache.num_tables, _p(r))


def generation_step(cache, alpha_h, alpha_l, window):
    """Algorithm 1 once for every table (after a decode step's append)."""
    st = cache.struct()
    lib().dko_generation_step(C.byref(cache.L), C.byref(st), float(alpha_h), float(alpha_l),
                              int(window))


def read_token(cache, t, sec, u):
    D = cache.L.head_dim
    k = np.zeros(D, np.float64)
    v = np.zeros(D, np.float64)
    s = np.zeros(1, np.float32)
    pos = np.zeros(1, np.int32)
    st = cache.struct()
    lib().dko_read_token(C.byref(cache.L), C.byref(st), t, sec, u, _p(k), _p(v), _p(s), _p(pos))
    return k, v, float(s[0]), int(pos[0])


def attention(cache, q, sm_scale):
    """q: fp16 bits uint16 [B][Hq][D].  Returns (out fp64 [B][Hq][D], lse fp64 [B][Hq])."""
    q = np.ascontiguousarray(q, np.uint16)
    B, Hq, D = q.shape
    out = np.zeros((B, Hq, D), np.float64)
    lse = np.zeros((B, Hq), np.float64)
    st = cache.struct()
    rc = lib().dko_attention(C.byref(cache.L), C.byref(st), Hq, _p(q), float(sm_scale),
                             _p(out), _p(lse))
    if rc != 0:
        raise ValueError("oracle: Hq must be a multiple of Hkv")
    return out, lse


def update_significance(cache, q, sm_scale):
    """One decode step's significance update of every kept token's score (in place)."""
    q = np.ascontiguousarray(q, np.uint16)
    st = cache.struct()
    if lib().dko_update_significance(C.byref(cache.L), C.byref(st), q.shape[1], _p(q), float(sm_scale)):
        raise ValueError("oracle: Hq must be a multiple of Hkv")


def prompt_significance(new_len, q, k, sm_scale, select=None, out=None):
    """Prompt-phase significance of every prompt token: q [rows][Hq][D], k [rows][Hkv][D]
    fp16 bits, rows concatenated per sequence; returns score [rows][Hkv] fp32.  With
    `select` ([B][Hkv] bool) only those tables are computed (others stay as in `out`)."""
    new_len = np.ascontiguousarray(new_len, np.int32)
    q = np.ascontiguousarray(q, np.uint16)
    k = np.ascontiguousarray(k, np.uint16)
    rows, Hq, D = q.shape
    Hkv = k.shape[1]
    assert k.shape == (rows, Hkv, D) and int(new_len.sum()) == rows
    score = np.zeros((rows, Hkv), np.float32) if out is None else out
    sel = None if select is None else np.ascontiguousarray(select, np.uint8)
    if lib().dko_prompt_significance(len(new_len), _p(new_len), Hq, Hkv, D, _p(q), _p(k), float(sm_scale),
                                     None if sel is None else _p(sel), _p(score)):
        raise ValueError("oracle: bad shapes")
    return score


def prompt_significance_tail(q, k, sm_scale, h, m):
    """Scores (fp64) of the last m tokens of one prompt (q [N][Hq][D], k [N][Hkv][D]
    fp16 bits) for KV head h."""
    q = np.ascontiguousarray(q, np.uint16)
    k = np.ascontiguousarray(k, np.uint16)
    N, Hq, D = q.shape
    out = np.zeros(m)
    if lib().dko_prompt_significance_tail(N, Hq, k.shape[1], D, _p(q), _p(k), float(sm_scale), int(h), int(m),
                                          _p(out)):
        raise ValueError("oracle: bad arguments")
    return out


def attention_partial(cache, q, sm_scale, b, hq, p0, p1):
    q = np.ascontiguousarray(q, np.uint16)
    Hq, D = q.shape[1], q.shape[2]
    m = np.zeros(1)
    l = np.zeros(1)
    acc = np.zeros(D)
    st = cache.struct()
    lib().dko_attention_partial(C.byref(cache.L), C.byref(st), Hq, _p(q), float(sm_scale),
                                b, hq, p0, p1, _p(m), _p(l), _p(acc))
    return float(m[0]), float(l[0]), acc


def merge_partials(m, l, acc):
    m = np.ascontiguousarray(m, np.float64)
    l = np.ascontiguousarray(l, np.float64)
    acc = np.ascontiguousarray(acc, np.float64)
    S, D = acc.shape
    out = np.zeros(D)
    lse = np.zeros(1)
    lib().dko_merge_partials(S, D, _p(m), _p(l), _p(acc), _p(out), _p(lse))
    return out, float(lse[0])


def kv_bits_fraction(L, n_hi, n_lo, n_total):
    kf = np.zeros(1)
    vf = np.zeros(1)
    lib().dko_kv_bits_fraction(C.byref(L), n_hi, n_lo, n_total, _p(kf), _p(vf))
    return float(kf[0]), float(vf[0])
