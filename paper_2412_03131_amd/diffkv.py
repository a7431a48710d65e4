"""Thin ctypes binding of libdiffkv.so (the C ABI declared in include/diffkv.h).

Argument marshalling only: every step of the hot path runs in the HIP
kernels of the library.  PyTorch provides device memory and the stream.
Loading fails loudly when the library has not been built.
"""
import ctypes as C
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libdiffkv.so")

OK, E_INVAL, E_UNSUPPORTED, E_WORKSPACE, E_LAUNCH, E_SCRATCH = 0, 1, 2, 3, 4, 5
ST_OUT_OF_PAGES, ST_TABLE_OVERFLOW, ST_BAD_INPUT = 1, 2, 4
OP_APPEND, OP_ATTENTION, OP_COMPACT, OP_ALLOC, OP_GENERATION, OP_PROMPT_SIGNIFICANCE = 0, 1, 2, 3, 4, 5
HIGH, LOW = 0, 1

_lib = None


class DiffKVError(RuntimeError):
    def __init__(self, code, what):
        super().__init__("%s: %s (status %d)" % (what, status_str(code), code))
        self.code = code


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


class CacheStruct(C.Structure):
    _fields_ = [
        ("pool", C.c_void_p), ("num_pages", C.c_int64),
        ("page_table", C.c_void_p), ("pages", C.c_void_p), ("len", C.c_void_p),
        ("seq_len", C.c_void_p), ("ring", C.c_void_p), ("ring_ptr", C.c_void_p),
        ("status", C.c_void_p), ("num_seqs", C.c_int32), ("num_kv_heads", C.c_int32),
    ]


EXPORTS = ("diffkv_layout_init", "diffkv_workspace_size", "diffkv_quantize_append",
           "diffkv_decode_attention", "diffkv_decode_attention_noalloc", "diffkv_update_significance",
           "diffkv_prompt_significance", "diffkv_compact_free_list", "diffkv_alloc_pages",
           "diffkv_generation_step", "diffkv_status_str")


def lib():
    """Load libdiffkv.so (raises if it is missing: there is no fallback path)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError("libdiffkv.so is not built (%s); run __graft_entry__.build()" % LIB_PATH)
        L = C.CDLL(LIB_PATH)
        vp, i32, i64, f32, sz = C.c_void_p, C.c_int32, C.c_int64, C.c_float, C.c_size_t
        PL = C.POINTER(Layout)
        PC = C.POINTER(CacheStruct)
        L.diffkv_layout_init.argtypes = [PL, i32, i32, vp, vp, vp, i32]
        L.diffkv_workspace_size.argtypes = [i32, PL, i32, i32, i32, i64, i32, C.POINTER(sz)]
        L.diffkv_quantize_append.argtypes = [PL, PC, i64, i32, vp, vp, vp, vp, vp, f32, f32, i32,
                                             vp, sz, vp]
        L.diffkv_decode_attention.argtypes = [PL, PC, i32, vp, f32, vp, vp, i32, vp, sz, vp]
        L.diffkv_decode_attention_noalloc.argtypes = [PL, PC, i32, vp, f32, vp, vp, i32, vp]
        L.diffkv_update_significance.argtypes = [PL, PC, i32, vp, f32, vp, vp]
        L.diffkv_prompt_significance.argtypes = [PL, i32, i64, i32, vp, i32, i32, vp, vp, f32, vp, vp,
                                                 vp, sz, vp]
        L.diffkv_compact_free_list.argtypes = [PL, PC, i32, vp, vp, sz, vp]
        L.diffkv_alloc_pages.argtypes = [PL, PC, i32, vp, vp, sz, vp]
        L.diffkv_generation_step.argtypes = [PL, PC, f32, f32, i32, vp, sz, vp]
        L.diffkv_status_str.argtypes = [i32]
        L.diffkv_status_str.restype = C.c_char_p
        for n in EXPORTS[:-1]:
            getattr(L, n).restype = i32
        _lib = L
    return _lib


def status_str(code):
    return lib().diffkv_status_str(code).decode()


def _check(code, what):
    if code != OK:
        raise DiffKVError(code, what)


def _ptr(t):
    return None if t is None else C.c_void_p(t.data_ptr())


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return C.c_void_p(stream.cuda_stream)


def layout(head_dim=128, group=32, k_bits=(8, 4), v_bits=(4, 2), tokens_per_page=(16, 32),
           max_seq_len=4096):
    L = Layout()
    kb = (C.c_int32 * 2)(*k_bits)
    vb = (C.c_int32 * 2)(*v_bits)
    tp = (C.c_int32 * 2)(*tokens_per_page)
    _check(lib().diffkv_layout_init(C.byref(L), head_dim, group, kb, vb, tp, max_seq_len),
           "diffkv_layout_init")
    return L


def workspace_size(op, L, num_seqs, num_q_heads=0, num_kv_heads=1, total_new=0, num_splits=0):
    n = C.c_size_t(0)
    _check(lib().diffkv_workspace_size(op, C.byref(L), num_seqs, num_q_heads, num_kv_heads,
                                       total_new, num_splits, C.byref(n)), "diffkv_workspace_size")
    return n.value


def _ws(nbytes, device, ws):
    if ws is not None:
        if ws.numel() * ws.element_size() < nbytes:
            raise ValueError("workspace too small: need %d bytes" % nbytes)
        return ws
    return torch.empty(max(nbytes, 256), dtype=torch.uint8, device=device)


class Cache:
    """Device tensors of one cache (diffkv_cache); the library owns none of them."""

    def __init__(self, L, num_pages, num_seqs, num_kv_heads, device="cuda", ring=None,
                 with_pool=True):
        self.L = L
        self.num_pages = int(num_pages)
        self.num_seqs = int(num_seqs)
        self.num_kv_heads = int(num_kv_heads)
        T = self.num_seqs * self.num_kv_heads
        dev = torch.device(device)
        self.pool = torch.zeros((self.num_pages if with_pool else 1, L.page_bytes),
                                dtype=torch.uint8, device=dev)
        self.page_table = torch.full((T, L.p_max), -1, dtype=torch.int32, device=dev)
        self.pages = torch.zeros((T, 2), dtype=torch.int32, device=dev)
        self.len = torch.zeros((T, 2), dtype=torch.int32, device=dev)
        self.seq_len = torch.zeros(self.num_seqs, dtype=torch.int32, device=dev)
        if ring is None:
            self.ring = torch.arange(self.num_pages, dtype=torch.int32, device=dev)
        else:
            self.ring = torch.as_tensor(ring, dtype=torch.int32).to(dev).contiguous()
        self.ring_ptr = torch.tensor([0, self.num_pages], dtype=torch.int64, device=dev)
        self.status = torch.zeros(1, dtype=torch.int32, device=dev)

    @property
    def num_tables(self):
        return self.num_seqs * self.num_kv_heads

    def view(self, seq_lo, seq_hi):
        """Cache over sequences [seq_lo, seq_hi) sharing this cache's pool, ring, pointers
        and status (e.g. one layer of a cache whose "sequences" are layer-major)."""
        v = Cache.__new__(Cache)
        v.L = self.L
        v.num_pages = self.num_pages
        v.num_seqs = seq_hi - seq_lo
        v.num_kv_heads = self.num_kv_heads
        H = self.num_kv_heads
        v.pool, v.ring, v.ring_ptr, v.status = self.pool, self.ring, self.ring_ptr, self.status
        v.page_table = self.page_table[seq_lo * H:seq_hi * H]
        v.pages = self.pages[seq_lo * H:seq_hi * H]
        v.len = self.len[seq_lo * H:seq_hi * H]
        v.seq_len = self.seq_len[seq_lo:seq_hi]
        return v

    def struct(self):
        return CacheStruct(self.pool.data_ptr(), self.num_pages, self.page_table.data_ptr(),
                           self.pages.data_ptr(), self.len.data_ptr(), self.seq_len.data_ptr(),
                           self.ring.data_ptr(), self.ring_ptr.data_ptr(), self.status.data_ptr(),
                           self.num_seqs, self.num_kv_heads)


def _bits16(t):
    return t if t.dtype in (torch.int16, torch.float16, torch.bfloat16) else t.view(torch.int16)


def quantize_append(cache, new_len, k, v, score, quota=None, alpha_h=0.0, alpha_l=0.0,
                    window=0, total_new=None, max_new=None, ws=None, stream=None):
    """new_len int32 [B] (device); k, v fp16 [total_new, Hkv, D]; score fp32 [total_new, Hkv];
    quota int32 [B, Hkv, 2] or None (threshold form).  total_new / max_new are host sizes
    (read from new_len with a device sync when omitted)."""
    L = cache.L
    if total_new is None or max_new is None:
        nl = new_len.cpu()
        total_new = int(nl.sum()) if total_new is None else total_new
        max_new = int(nl.max()) if max_new is None else max_new
    need = workspace_size(OP_APPEND, L, cache.num_seqs, 0, cache.num_kv_heads, total_new)
    ws = _ws(need, cache.pool.device, ws)
    st = cache.struct()
    _check(lib().diffkv_quantize_append(
        C.byref(L), C.byref(st), int(total_new), int(max_new), _ptr(new_len), _ptr(_bits16(k)),
        _ptr(_bits16(v)), _ptr(score), _ptr(quota), float(alpha_h), float(alpha_l), int(window),
        _ptr(ws), ws.numel() * ws.element_size(), _stream(stream)), "diffkv_quantize_append")
    return ws


def decode_attention(cache, q, sm_scale, out=None, lse=None, num_splits=0, ws=None, stream=None,
                     want_lse=True):
    """q fp16 [B, Hq, D] (device) -> out fp32 [B, Hq, D], lse fp32 [B, Hq]."""
    L = cache.L
    B, Hq, D = q.shape
    if out is None:
        out = torch.empty((B, Hq, D), dtype=torch.float32, device=q.device)
    if lse is None and want_lse:
        lse = torch.empty((B, Hq), dtype=torch.float32, device=q.device)
    need = workspace_size(OP_ATTENTION, L, cache.num_seqs, Hq, cache.num_kv_heads, 0, num_splits)
    ws = _ws(need, q.device, ws)
    st = cache.struct()
    _check(lib().diffkv_decode_attention(
        C.byref(L), C.byref(st), Hq, _ptr(_bits16(q)), float(sm_scale), _ptr(out), _ptr(lse),
        int(num_splits), _ptr(ws), ws.numel() * ws.element_size(), _stream(stream)),
        "diffkv_decode_attention")
    return out, lse


def decode_attention_noalloc(cache, q, sm_scale, out, lse=None, num_splits=0, stream=None):
    """diffkv_decode_attention_noalloc: like decode_attention, outputs given by the
    caller, no workspace (the library's fixed per-device scratch)."""
    st = cache.struct()
    _check(lib().diffkv_decode_attention_noalloc(
        C.byref(cache.L), C.byref(st), q.shape[1], _ptr(_bits16(q)), float(sm_scale), _ptr(out),
        _ptr(lse), int(num_splits), _stream(stream)), "diffkv_decode_attention_noalloc")
    return out, lse


def update_significance(cache, q, sm_scale, lse, stream=None):
    """diffkv_update_significance: every kept token's score becomes the running mean of
    its attention probability (max over the KV head's query heads); lse from
    decode_attention with the same q."""
    st = cache.struct()
    _check(lib().diffkv_update_significance(C.byref(cache.L), C.byref(st), q.shape[1], _ptr(_bits16(q)),
                                            float(sm_scale), _ptr(lse), _stream(stream)),
           "diffkv_update_significance")


def prompt_significance(L, new_len, q, k, sm_scale, lse=None, score=None, max_new=None, ws=None,
                        stream=None):
    """diffkv_prompt_significance: q fp16 [rows, Hq, D], k fp16 [rows, Hkv, D] (device, rows
    concatenated per sequence), new_len int32 [B] (device); returns score fp32 [rows, Hkv].
    lse (fp32 [rows, Hq], natural log) skips the row pass when given."""
    rows, Hq, Hkv = q.shape[0], q.shape[1], k.shape[1]
    B = new_len.shape[0]
    if max_new is None:
        max_new = int(new_len.max().item()) if B else 0
    if score is None:
        score = torch.empty((rows, Hkv), dtype=torch.float32, device=q.device)
    need = workspace_size(OP_PROMPT_SIGNIFICANCE, L, B, Hq, Hkv, rows)
    ws = _ws(need, q.device, ws)
    _check(lib().diffkv_prompt_significance(C.byref(L), B, rows, int(max_new), _ptr(new_len), Hq, Hkv,
                                            _ptr(_bits16(q)), _ptr(_bits16(k)), float(sm_scale), _ptr(lse),
                                            _ptr(score), _ptr(ws), ws.numel() * ws.element_size(),
                                            _stream(stream)), "diffkv_prompt_significance")
    return score


def compact_free_list(cache, release, num_tables=None, ws=None, stream=None):
    """release uint8 [num_tables, p_max] (device)."""
    L = cache.L
    nt = cache.num_tables if num_tables is None else num_tables
    need = workspace_size(OP_COMPACT, L, cache.num_seqs, 0, cache.num_kv_heads)
    ws = _ws(need, cache.pool.device, ws)
    st = cache.struct()
    _check(lib().diffkv_compact_free_list(C.byref(L), C.byref(st), int(nt), _ptr(release),
                                          _ptr(ws), ws.numel() * ws.element_size(),
                                          _stream(stream)), "diffkv_compact_free_list")
    return ws


def alloc_pages(cache, demand, num_tables=None, ws=None, stream=None):
    """demand int32 [num_tables, 2] (device)."""
    L = cache.L
    nt = cache.num_tables if num_tables is None else num_tables
    need = workspace_size(OP_ALLOC, L, cache.num_seqs, 0, cache.num_kv_heads)
    ws = _ws(need, cache.pool.device, ws)
    st = cache.struct()
    _check(lib().diffkv_alloc_pages(C.byref(L), C.byref(st), int(nt), _ptr(demand), _ptr(ws),
                                    ws.numel() * ws.element_size(), _stream(stream)),
           "diffkv_alloc_pages")
    return ws


def generation_step(cache, alpha_h, alpha_l, recent_window, ws=None, stream=None):
    """One decode step's generation-phase policy for every table (Algorithm 1)."""
    L = cache.L
    need = workspace_size(OP_GENERATION, L, cache.num_seqs, 0, cache.num_kv_heads)
    ws = _ws(need, cache.pool.device, ws)
    st = cache.struct()
    _check(lib().diffkv_generation_step(C.byref(L), C.byref(st), float(alpha_h), float(alpha_l),
                                        int(recent_window), _ptr(ws),
                                        ws.numel() * ws.element_size(), _stream(stream)),
           "diffkv_generation_step")
    return ws
