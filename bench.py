#!/usr/bin/env python3
"""Benchmark of the DiffKV decode hot path on one MI355X.

Headline workload (--config long32k, the default): the long-generation shape, batch 16,
40 query / 8 KV heads (GQA 5:1), head_dim 128, 32768-token contexts whose per-head pruned
fraction is 0.1 + 0.8 * Beta(2, 2) and whose kept tokens are split evenly between K8V4 and
K4V2 (group-32 fp16 scale/zero, 16/32 tokens per page).  The prompt phase fills the cache
(one diffkv_quantize_append), then every timed step is one decode step of the path:

  1. diffkv_quantize_append of one new token per (sequence, KV head), quota (1, 0): the
     token enters the recent window at high precision (classing, allocation when a page
     fills, quantization, placement);
  2. diffkv_decode_attention over the whole compressed cache (automatic split mode).

value = KV tokens attended per second of step time (a KV token is one kept
(token, KV head) pair), from the wall clock around K back-to-back steps.  A second pass of
K steps evicts the Infinity Cache and L2 before every step (a reduction reading 1 GiB,
outside the HIP events) and gives the per-launch attention and append times (median, p10, p90,
mean) and the roofline: algorithmic compressed bytes / mean attention time.

Extra keys of the same JSON line:
  significance    the decode step's significance update (running mean of each kept
                  token's attention probability, Sec. 4) on the headline cache;
  precisions      attention time per precision level (K8V8 .. K4V1) against its KV bytes;
  llama70b        batch 32, 64 query / 8 KV heads (GQA 8:1), context 8192, split 30/40/30:
                  attention with num_splits = 1 (no split), automatic, and balanced
                  shares + merge (sequence split), each timed after a cache flush;
  serving_step    the llama8b shape (batch 64, 32/8 heads, contexts U[1024, 4096]) on four
                  layers sharing one pool: per step one request finishes (one compaction
                  call for all layers), a new request is prefilled while the other 63
                  decode (one append call for all layers), then attention per layer;
  compaction      2^20-page pool, 4096 tables, 100 rounds of Bernoulli(0.35) releases;
  generation_step the generation-phase policy (Algorithm 1) per decode step, llama8b;
  memory_management  compaction + allocation per step at context 1024 for batches 8/32/128
                  (32 layers x 8 KV heads per request) on the GPU and on a 16-thread host
                  memory manager (baselines/cpu_manager.c), states checked identical;
  cpu_baseline    the CPU oracle's fp64 attention on a bounded sample of the headline
                  workload, one thread and all host cores (threads; the oracle's C code
                  releases the interpreter lock), plus its serial compaction.
"""
import argparse
import ctypes as C
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "decode-attention KV tokens/s + achieved HBM GB/s (% of peak); compaction pages/s"
HBM_PEAK_GBPS = 8000.0
SCALE = 1.0 / np.sqrt(128.0)
ATTN_SOURCES = ["k_attention.hip", "attn_kernels.hpp", "attn_common.hpp", "k_attn_l0.hip", "internal.hpp",
                "common.hpp"]
FLUSH_BYTES = 1 << 30   # > the 256 MB Infinity Cache + 8 x 4 MB L2
DTYPE_DETAIL = ("q.k: fp16 q x integer codes (exact products), fp32 sums, fp32 scale/zero; "
                "p.v: softmax weight x fp16 scale rounded to fp16 x integer codes, fp32 sums; "
                "softmax, merge and outputs fp32")

WORKLOADS = {
    "long32k": "long-generation decode step: B=16, Hq=40, Hkv=8 (GQA 5), D=128, context 32768, "
               "pruned fraction 0.1+0.8*Beta(2,2) per head, kept tokens half K8V4 half K4V2, group 32, "
               "16/32 tokens per page; per step one 1-token quantize_append per (sequence, KV head) "
               "then attention over the whole cache",
    "llama70b": "Llama-3-70B-shaped decode step: B=32, Hq=64, Hkv=8 (GQA 8), D=128, context 8192, "
                "high/low/pruned 30/40/30 per head, group 32, 16/32 tokens per page; per step one "
                "1-token quantize_append per (sequence, KV head) then attention",
    "llama8b": "Llama-3-8B-shaped decode step: B=64, Hq=32, Hkv=8 (GQA 4), D=128, context U[1024,4096], "
               "f_hi U[0.1,0.5], f_pr U[0.2,0.6], group 32, 16/32 tokens per page; per step one "
               "1-token quantize_append per (sequence, KV head) then attention",
}


def traffic_file(config):
    return os.path.join(ROOT, "profiles", "attn_%s_traffic.txt" % config)


def attention_sources_sha256():
    import hashlib
    h = hashlib.sha256()
    for f in ATTN_SOURCES:
        with open(os.path.join(ROOT, "paper_2412_03131_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def measured_traffic(config):
    """HBM bytes per attention launch from the committed counter summary of this
    workload, or None when it is missing or was taken on different attention sources."""
    try:
        kv = {}
        with open(traffic_file(config)) as fh:
            for ln in fh:
                if ":" in ln and not ln.startswith("#"):
                    k, v = ln.split(":", 1)
                    kv[k.strip()] = v.strip()
        if kv.get("sources_sha256") != attention_sources_sha256():
            return None
        return float(kv["traffic_bytes_per_launch"])
    except (OSError, KeyError, ValueError):
        return None


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=64, help="timed decode steps (per pass)")
    ap.add_argument("--warmup", type=int, default=320,
                    help="untimed warm-up iterations: W - min(W, 8) attention calls on the prompt's cache, "
                         "then min(W, 8) full decode steps (back-to-back steps reach their steady time only "
                         "after ~25 ms of work: 110 us per long32k step after 64 full warm-up steps, 97-99 "
                         "after 320)")
    ap.add_argument("--config", choices=("long32k", "llama70b", "llama8b"), default="long32k",
                    help="headline decode workload")
    ap.add_argument("--splits", type=int, default=0,
                    help="attention mode: 0 automatic, -1 balanced shares, S >= 1 ranges per table")
    ap.add_argument("--extras", choices=("all", "none"), default="all",
                    help="'none' prints the headline line only (no llama70b modes, serving step, "
                         "compaction, generation step)")
    ap.add_argument("--serving-steps", type=int, default=30)
    ap.add_argument("--layers", type=int, default=4, help="layers of the serving step")
    ap.add_argument("--reps", type=int, default=40, help="flushed attention calls per llama70b mode")
    ap.add_argument("--compaction-rounds", type=int, default=100)
    ap.add_argument("--generation-steps", type=int, default=50)
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--only", choices=("all", "attention", "copy", "generation", "prompt", "compaction"),
                    default="all",
                    help="profiling aids that print no benchmark line: 'attention' builds the "
                         "--config cache and times only attention calls (no flush); 'copy' runs a "
                         "plain 1 GiB device copy (the reference for scaling HBM byte counters); "
                         "'generation' runs only the generation-step measurement; 'prompt' only "
                         "the prompt-phase significance measurement; 'compaction' only the "
                         "compaction workload")
    return ap.parse_args()


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


def attn_bytes(len_hi, len_lo, B, Hq, Hkv):
    """Algorithmic bytes of one attention launch: compressed K/V codes + fp16 scale/zero
    (224 B per high token, 128 B per low token), the table entries of the used pages,
    the section lengths, q in, out and lse."""
    ph = -(-len_hi // 16)
    pl = -(-len_lo // 32)
    kv = 224 * int(len_hi.sum()) + 128 * int(len_lo.sum())
    return kv + 4 * int(ph.sum() + pl.sum()) + 8 * len_hi.size + B * Hq * 128 * (2 + 4) + 4 * B * Hq


def pct(a):
    a = np.asarray(a, np.float64)
    return {"mean": float(a.mean()), "median": float(np.median(a)),
            "p10": float(np.percentile(a, 10)), "p90": float(np.percentile(a, 90))}


def to_dev(torch, dev, a):
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        a = a.view(np.int16)
    return torch.from_numpy(a).to(dev)


class HipEvent:
    """A HIP timing event recorded on the launch stream without system-scope fences
    (hipEventDisableSystemFence).  An event of the default kind (what torch.cuda.Event
    creates) records with a system-scope release and acquire; measured on MI355X, each
    such record delays the next launch on the stream by 5.7 us, against 4.4 us for
    this kind (the marker itself), and that delay falls inside the timed interval.
    The stream stays in order: the record still waits for the work before it.  Same
    interface as torch.cuda.Event: record(), elapsed_time(end) in ms."""
    hip = None
    stream = None

    @classmethod
    def setup(cls, stream_ptr):
        """Bind to the HIP runtime that torch loaded (the one libdiffkv.so links to) and
        to the stream the library launches on; call after torch has initialised HIP."""
        path = None
        with open("/proc/self/maps") as f:
            for line in f:
                if "libamdhip64.so" in line:
                    path = line.split()[-1]
                    break
        if path is None:
            raise RuntimeError("the HIP runtime is not loaded")
        cls.hip = C.CDLL(path)
        cls.hip.hipEventCreateWithFlags.argtypes = [C.POINTER(C.c_void_p), C.c_uint]
        cls.hip.hipEventRecord.argtypes = [C.c_void_p, C.c_void_p]
        cls.hip.hipEventElapsedTime.argtypes = [C.POINTER(C.c_float), C.c_void_p, C.c_void_p]
        cls.stream = stream_ptr

    def __init__(self):
        self.e = C.c_void_p()
        self._check(self.hip.hipEventCreateWithFlags(C.byref(self.e), 0x20000000), "create")

    @staticmethod
    def _check(rc, what):
        if rc != 0:
            raise RuntimeError("hipEvent %s failed (%d)" % (what, rc))

    def record(self):
        self._check(self.hip.hipEventRecord(self.e, self.stream), "record")

    def elapsed_time(self, end):
        ms = C.c_float()
        self._check(self.hip.hipEventElapsedTime(C.byref(ms), self.e, end.e), "elapsed time")
        return ms.value


class Flush:
    """Evicts the Infinity Cache and the L2s with clean lines: a reduction that reads
    1 GiB.  (A fill kernel would leave dirty lines whose write-back then lands inside
    the next timed launch: measured +27 us on a 43 us llama8b call.)"""

    def __init__(self, torch, dev):
        self.torch = torch
        self.buf = torch.zeros(FLUSH_BYTES // 4, dtype=torch.int32, device=dev)
        self.out = torch.zeros(1, dtype=torch.int64, device=dev)

    def __call__(self):
        self.torch.sum(self.buf, dim=(0,), dtype=self.torch.int64, out=self.out[0])


def build_decode(torch, dk, dev, name, extra_steps):
    """Prompt phase of a decode workload on the GPU; per-step decode inputs for
    `extra_steps` steps (one token per sequence, quota (1, 0))."""
    from paper_2412_03131_amd import inputs
    t0 = time.time()
    w = inputs.prefill(name)
    B, Hq, Hkv = w["B"], w["Hq"], w["Hkv"]
    nl = w["new_len"].astype(np.int64)
    hi0 = w["quota"][:, :, 0].astype(np.int64)
    lo0 = w["quota"][:, :, 1].astype(np.int64)
    L = dk.layout(max_seq_len=int(nl.max()) + extra_steps + 16)
    per_table = (-(-(hi0 + extra_steps) // 16)) + (-(-lo0 // 32)) + 2
    num_pages = int(per_table.sum()) + 256
    cache = dk.Cache(L, num_pages, B, Hkv, device=dev)
    T = lambda a: to_dev(torch, dev, a)
    dk.quantize_append(cache, T(w["new_len"]), T(w["k"]), T(w["v"]), T(w["score"]), quota=T(w["quota"]),
                       total_new=int(nl.sum()), max_new=int(nl.max()))
    torch.cuda.synchronize()
    if int(cache.status.item()) != 0:
        raise RuntimeError("prefill raised status %d" % int(cache.status.item()))
    steps = []
    for s in range(extra_steps):
        d = inputs.decode_token(name, s, B, Hq, Hkv, w["outliers"])
        steps.append(dict(k=T(d["k"]), v=T(d["v"]), score=T(d["score"]), quota=T(d["quota"]), q=T(d["q"])))
    log("workload %s: B=%d Hq=%d Hkv=%d, %d prompt rows, %d pages (%.2f GB pool), built in %.1f s"
        % (name, B, Hq, Hkv, int(nl.sum()), num_pages, num_pages * L.page_bytes / 1e9, time.time() - t0))
    res = dict(w=dict(B=B, Hq=Hq, Hkv=Hkv, new_len=w["new_len"], quota=w["quota"]), L=L, cache=cache,
               steps=steps, hi0=hi0.reshape(-1), lo0=lo0.reshape(-1), ones=T(np.ones(B, np.int32)))
    del w
    return res


def decode_headline(torch, dk, lib, dev, sptr, wl, args, flush):
    """K back-to-back decode steps (the contract's timed region, no instrumentation
    inside it: HIP events between back-to-back calls add GPU-side gaps, measured
    about 16 us per step), then K steps after cache eviction timed per launch with
    HIP events on the launch stream (the roofline figures), then K back-to-back steps
    with events (unflushed per-launch times, for reference)."""
    B, Hq, Hkv = wl["w"]["B"], wl["w"]["Hq"], wl["w"]["Hkv"]
    L, cache = wl["L"], wl["cache"]
    S = args.splits
    out = torch.empty((B, Hq, 128), dtype=torch.float32, device=dev)
    lse = torch.empty((B, Hq), dtype=torch.float32, device=dev)
    ws_att = torch.empty(max(256, dk.workspace_size(dk.OP_ATTENTION, L, B, Hq, Hkv, 0, S)),
                         dtype=torch.uint8, device=dev)
    ws_app = torch.empty(dk.workspace_size(dk.OP_APPEND, L, B, 0, Hkv, B) + 256, dtype=torch.uint8, device=dev)
    Lp = C.byref(L)
    cs = cache.struct()
    vp = lambda x: C.c_void_p(x.data_ptr())
    app, att = [], []
    for si in wl["steps"]:
        app.append((Lp, C.byref(cs), B, 1, vp(wl["ones"]), vp(si["k"]), vp(si["v"]), vp(si["score"]),
                    vp(si["quota"]), 0.0, 0.0, 0, vp(ws_app), ws_app.numel(), sptr))
        att.append((Lp, C.byref(cs), Hq, vp(si["q"]), float(SCALE), vp(out), vp(lse), S, vp(ws_att),
                    ws_att.numel(), sptr))
    K, W = args.steps, args.warmup
    # warm-up: W - F attention calls on the cache as the prompt left it (they bring
    # the GPU to its steady clock without growing the cache), then F full steps
    F = min(W, 8)
    ev = [[HipEvent() for _ in range(3)] for _ in range(2 * K)]  # passes 2, 3

    def step(s, e=None):
        if e is not None:
            e[0].record()
        rc = lib.diffkv_quantize_append(*app[s])
        if e is not None:
            e[1].record()
        rc |= lib.diffkv_decode_attention(*att[s])
        if e is not None:
            e[2].record()
        if rc:
            raise RuntimeError("library call failed at step %d (rc %d)" % (s, rc))

    # expected section lengths at every step's attention (bytes and token counts)
    hi, lo = wl["hi0"].copy(), wl["lo0"].copy()
    step_bytes, step_tok = [], []
    for s in range(F + 3 * K):
        hi = hi + 1
        step_bytes.append(attn_bytes(hi, lo, B, Hq, Hkv))
        step_tok.append(int(hi.sum() + lo.sum()))
    for s in range(W - F):
        if lib.diffkv_decode_attention(*att[0]):
            raise RuntimeError("library call failed in the warm-up")
    for s in range(F):
        step(s)
    torch.cuda.synchronize()
    # pass 1: the timed region of the contract, back to back
    t0 = time.perf_counter()
    for i in range(K):
        step(F + i)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    # pass 2: caches evicted before every step (outside the events)
    for i in range(K):
        flush()
        step(F + K + i, ev[i])
    torch.cuda.synchronize()
    # pass 3: back to back with events
    for i in range(K):
        step(F + 2 * K + i, ev[K + i])
    torch.cuda.synchronize()
    status = int(cache.status.item())
    got = cache.len.cpu().numpy()
    if status != 0 or not (np.array_equal(got[:, 0], hi) and np.array_equal(got[:, 1], lo)):
        raise RuntimeError("state check failed after the timed steps (status %d)" % status)
    app_us = np.array([e[0].elapsed_time(e[1]) * 1e3 for e in ev])
    att_us = np.array([e[1].elapsed_time(e[2]) * 1e3 for e in ev])
    tok1 = np.array(step_tok[F:F + K], np.float64)
    byt2 = np.array(step_bytes[F + K:F + 2 * K], np.float64)
    tok2 = np.array(step_tok[F + K:F + 2 * K], np.float64)
    byt3 = np.array(step_bytes[F + 2 * K:], np.float64)
    a2, p2 = att_us[:K], app_us[:K]
    a3, p3 = att_us[K:], app_us[K:]
    achieved = float(byt2.sum() / (a2.sum() * 1e-6) / 1e9)
    res = dict(
        value=float(tok1.sum() / wall), wall=wall, ms_per_step=wall / K * 1e3,
        achieved=achieved, bytes_per_launch=float(byt2.mean()), us_per_launch=float(a2.mean()),
        attention=dict(flushed_us=pct(a2), flushed_gbps=achieved,
                       unflushed_us=pct(a3),
                       unflushed_gbps=float(byt3.sum() / (a3.sum() * 1e-6) / 1e9),
                       kv_tokens_per_launch=float(tok2.mean()),
                       kv_tokens_per_s=float(tok2.sum() / (a2.sum() * 1e-6)),
                       fp16_equivalent_gbps=float(tok2.sum() * 512 / (a2.sum() * 1e-6) / 1e9),
                       bytes_per_launch=float(byt2.mean())),
        append=dict(flushed_us=pct(p2), unflushed_us=pct(p3), tokens_per_call=B * Hkv),
        step=dict(flushed_us=pct(a2 + p2), unflushed_us=pct(a3 + p3),
                  back_to_back_us=wall / K * 1e6))
    log("headline: %.3f ms/step (wall, back to back), attention %.1f us/launch flushed (median %.1f, "
        "p10 %.1f, p90 %.1f), %.0f GB/s; unflushed %.1f us; append %.1f us"
        % (res["ms_per_step"], a2.mean(), np.median(a2), np.percentile(a2, 10), np.percentile(a2, 90),
           achieved, a3.mean(), p2.mean()))
    return res


def attention_modes(torch, dk, lib, dev, sptr, wl, reps, flush, modes=(1, 0, -1)):
    """Flushed attention calls over a built cache in several split modes."""
    B, Hq, Hkv = wl["w"]["B"], wl["w"]["Hq"], wl["w"]["Hkv"]
    L, cache = wl["L"], wl["cache"]
    lens = cache.len.cpu().numpy()
    nbytes = attn_bytes(lens[:, 0].astype(np.int64), lens[:, 1].astype(np.int64), B, Hq, Hkv)
    ntok = int(lens.sum())
    q = wl["steps"][0]["q"]
    out = torch.empty((B, Hq, 128), dtype=torch.float32, device=dev)
    lse = torch.empty((B, Hq), dtype=torch.float32, device=dev)
    res = {}
    for S in modes:
        ws = torch.empty(max(256, dk.workspace_size(dk.OP_ATTENTION, L, B, Hq, Hkv, 0, S)),
                         dtype=torch.uint8, device=dev)
        args = (C.byref(L), C.byref(cache.struct()), Hq, C.c_void_p(q.data_ptr()), float(SCALE),
                C.c_void_p(out.data_ptr()), C.c_void_p(lse.data_ptr()), S, C.c_void_p(ws.data_ptr()),
                ws.numel(), sptr)
        for _ in range(5):
            lib.diffkv_decode_attention(*args)
        ev = [(HipEvent(), HipEvent()) for _ in range(reps)]
        rc = 0
        for e in ev:
            flush()
            e[0].record()
            rc |= lib.diffkv_decode_attention(*args)
            e[1].record()
        torch.cuda.synchronize()
        if rc:
            raise RuntimeError("attention call failed (mode %d)" % S)
        us = np.array([a.elapsed_time(b) * 1e3 for a, b in ev])
        name = {1: "splits_1", 0: "automatic", -1: "balanced"}.get(S, "splits_%d" % S)
        gbps = nbytes / (us.mean() * 1e-6) / 1e9
        res[name] = dict(num_splits=S, us=pct(us), gbps=gbps, frac=gbps / HBM_PEAK_GBPS,
                         kv_tokens_per_s=ntok / (us.mean() * 1e-6))
        log("  attention mode %s: %.1f us (median %.1f, p10 %.1f, p90 %.1f), %.0f GB/s"
            % (name, us.mean(), np.median(us), np.percentile(us, 10), np.percentile(us, 90), gbps))
    res["bytes_per_launch"] = nbytes
    res["kv_tokens_per_launch"] = ntok
    return res


def significance_bench(torch, dk, lib, dev, sptr, wl, flush, reps=30):
    """diffkv_update_significance on the headline cache, right after each attention
    call with the same q (as a decode step runs it), caches evicted before the
    attention.  Algorithmic bytes: key codes and metadata (144 B per high token, 80 B
    per low token), the score read and written and the position read (12 B), the
    used table entries, q and lse."""
    B, Hq, Hkv = wl["w"]["B"], wl["w"]["Hq"], wl["w"]["Hkv"]
    L, cache = wl["L"], wl["cache"]
    lens = cache.len.cpu().numpy().astype(np.int64)
    hi, lo = lens[:, 0], lens[:, 1]
    nbytes = (156 * int(hi.sum()) + 92 * int(lo.sum()) + 4 * int((-(-hi // 16)).sum() + (-(-lo // 32)).sum())
              + B * Hq * (2 * 128 + 4))
    abytes = attn_bytes(hi, lo, B, Hq, Hkv)
    q = wl["steps"][0]["q"]
    out = torch.empty((B, Hq, 128), dtype=torch.float32, device=dev)
    lse = torch.empty((B, Hq), dtype=torch.float32, device=dev)
    ws = torch.empty(max(256, dk.workspace_size(dk.OP_ATTENTION, L, B, Hq, Hkv, 0, 0)), dtype=torch.uint8, device=dev)
    cs = cache.struct()
    att = (C.byref(L), C.byref(cs), Hq, C.c_void_p(q.data_ptr()), float(SCALE), C.c_void_p(out.data_ptr()),
           C.c_void_p(lse.data_ptr()), 0, C.c_void_p(ws.data_ptr()), ws.numel(), sptr)
    upd = (C.byref(L), C.byref(cs), Hq, C.c_void_p(q.data_ptr()), float(SCALE), C.c_void_p(lse.data_ptr()), sptr)
    ev = [[HipEvent() for _ in range(3)] for _ in range(reps)]
    ev2 = [[HipEvent() for _ in range(2)] for _ in range(reps)]
    rc = 0
    for _ in range(3):
        rc |= lib.diffkv_decode_attention(*att)
        rc |= lib.diffkv_update_significance(*upd)
    for e in ev:
        flush()
        e[0].record()
        rc |= lib.diffkv_decode_attention(*att)
        e[1].record()
        rc |= lib.diffkv_update_significance(*upd)
        e[2].record()
    for e in ev2:   # the update alone, caches evicted before it
        flush()
        e[0].record()
        rc |= lib.diffkv_update_significance(*upd)
        e[1].record()
    torch.cuda.synchronize()
    if rc:
        raise RuntimeError("significance bench: call failed")
    a_us = np.array([x[0].elapsed_time(x[1]) * 1e3 for x in ev])
    u_us = np.array([x[1].elapsed_time(x[2]) * 1e3 for x in ev])
    c_us = np.array([x[0].elapsed_time(x[1]) * 1e3 for x in ev2])
    res = {"workload": "the headline cache after its timed steps; per rep: cache eviction, attention, "
                       "then the significance update with the attention's lse",
           "us": pct(u_us), "attention_us": pct(a_us), "us_alone_flushed": pct(c_us),
           "bytes_per_launch": nbytes, "gbps": nbytes / (u_us.mean() * 1e-6) / 1e9,
           "bytes_vs_attention": nbytes / abytes, "time_vs_attention": float(u_us.mean() / a_us.mean())}
    log("significance update: %.1f us after a %.1f us attention call, %.1f us alone after eviction "
        "(%.2f of the attention's bytes)" % (u_us.mean(), a_us.mean(), c_us.mean(), nbytes / abytes))
    return res


MFMA_F16_PEAK = 2.5e15   # dense fp16 matrix-core peak of the MI355X, FLOP/s


def prompt_significance_bench(torch, dk, lib, dev, sptr, reps=5):
    """diffkv_prompt_significance over the llama8b prompt batch (B=64, Hq=32, Hkv=8,
    prompts of 1024-4096 tokens), with the row pass (no lse given) and without it (the
    row normalizers passed in, as a prompt attention kernel would supply them).
    Algorithmic FLOPs per pass: 2 * 128 per causal (query head, query, key) triple."""
    from paper_2412_03131_amd import inputs
    w = inputs.prefill("llama8b")
    B, Hq, Hkv = w["B"], w["Hq"], w["Hkv"]
    nl = w["new_len"].astype(np.int64)
    rows = int(nl.sum())
    q = torch.from_numpy(inputs.prompt_queries("llama8b", rows).view(np.int16)).to(dev).view(torch.float16)
    k = torch.from_numpy(w["k"].view(np.int16)).to(dev).view(torch.float16)
    new_len = torch.from_numpy(w["new_len"].astype(np.int32)).to(dev)
    L = dk.layout(max_seq_len=64)
    score = torch.empty((rows, Hkv), dtype=torch.float32, device=dev)
    ws = torch.empty(dk.workspace_size(dk.OP_PROMPT_SIGNIFICANCE, L, B, Hq, Hkv, rows), dtype=torch.uint8,
                     device=dev)
    lse = torch.zeros((rows, Hq), dtype=torch.float32, device=dev)
    vp = lambda x: C.c_void_p(x.data_ptr())
    call = lambda l: lib.diffkv_prompt_significance(C.byref(L), B, rows, int(nl.max()), vp(new_len), Hq, Hkv,
                                                    vp(q), vp(k), float(SCALE), l, vp(score), vp(ws),
                                                    ws.numel(), sptr)
    rc = call(None) | call(None)
    # (the normalizers passed in are zeros: their values do not change the work)
    ev = [[HipEvent() for _ in range(3)] for _ in range(reps)]
    for e in ev:
        e[0].record()
        rc |= call(None)
        e[1].record()
        rc |= call(vp(lse))
        e[2].record()
    torch.cuda.synchronize()
    if rc:
        raise RuntimeError("prompt significance bench: call failed")
    pairs = int((Hq * nl * (nl + 1) // 2).sum())
    flop_pass = 2.0 * 128 * pairs
    full = np.array([e[0].elapsed_time(e[1]) * 1e3 for e in ev])
    cols = np.array([e[1].elapsed_time(e[2]) * 1e3 for e in ev])
    res = {"workload": "llama8b prompt batch: B=64, Hq=32, Hkv=8 (GQA 4), D=128, prompts of 1024-4096 "
                       "tokens (%d rows), fp16 q/k" % rows,
           "us_both_passes": pct(full), "us_column_pass_lse_given": pct(cols),
           "flop_per_pass": flop_pass,
           "tflops_both_passes": 2 * flop_pass / (full.mean() * 1e-6) / 1e12,
           "tflops_column_pass": flop_pass / (cols.mean() * 1e-6) / 1e12,
           "frac_of_mfma_f16_peak_both": 2 * flop_pass / (full.mean() * 1e-6) / MFMA_F16_PEAK,
           "frac_of_mfma_f16_peak_column": flop_pass / (cols.mean() * 1e-6) / MFMA_F16_PEAK}
    log("prompt significance (llama8b prompts, %d rows): %.0f us both passes (%.0f TFLOP/s, %.2f of the "
        "fp16 MFMA peak), %.0f us column pass alone (%.0f TFLOP/s)"
        % (rows, full.mean(), res["tflops_both_passes"], res["frac_of_mfma_f16_peak_both"], cols.mean(),
           res["tflops_column_pass"]))
    return res


PRECISIONS = [  # (name, layout keyword arguments, section holding every token)
    ("K8V8", dict(k_bits=(8, 4), v_bits=(8, 2), tokens_per_page=(16, 32)), 0),
    ("K8V4", dict(k_bits=(8, 4), v_bits=(4, 2), tokens_per_page=(16, 32)), 0),
    ("K8V2", dict(k_bits=(8, 4), v_bits=(2, 1), tokens_per_page=(16, 32)), 0),
    ("K4V2", dict(k_bits=(8, 4), v_bits=(4, 2), tokens_per_page=(16, 32)), 1),
    ("K4V2/16", dict(k_bits=(8, 4), v_bits=(4, 2), tokens_per_page=(16, 16)), 1),
    ("K4V1", dict(k_bits=(8, 4), v_bits=(2, 1), tokens_per_page=(16, 32)), 1),
]


def precision_bench(torch, dk, lib, dev, sptr, flush, B=64, Hq=32, Hkv=8, L=2048, reps=20):
    """Attention time per precision level against its KV bytes, the shape of the
    paper's kernel speedup that follows the KV-size reduction (Sec. 7.3): the llama8b
    decode shape with L = 2048 tokens per sequence, no pruning, every token at one
    precision (one section of a layout), caches evicted before each call."""
    from paper_2412_03131_amd import inputs
    w = inputs.uniform_cache(B, Hq, Hkv, L)
    T = lambda a: to_dev(torch, dev, a)
    k, v, score, q, nl = T(w["k"]), T(w["v"]), T(w["score"]), T(w["q"]), T(w["new_len"])
    res = {"workload": "B=%d, Hq=%d, Hkv=%d, %d tokens per sequence, no pruning, every token at the "
                       "named precision; flushed attention calls" % (B, Hq, Hkv, L), "levels": {}}
    ntok = B * Hkv * L
    for name, kw, sec in PRECISIONS:
        Ld = dk.layout(max_seq_len=L + 16, **kw)
        Tp = kw["tokens_per_page"][sec]
        npg = B * Hkv * (-(-L // Tp)) + 64
        c = dk.Cache(Ld, npg, B, Hkv, device=dev)
        quota = np.zeros((B, Hkv, 2), np.int32)
        quota[:, :, sec] = L
        dk.quantize_append(c, nl, k, v, score, quota=T(quota), total_new=B * L, max_new=L)
        ws = torch.empty(max(256, dk.workspace_size(dk.OP_ATTENTION, Ld, B, Hq, Hkv, 0, 0)), dtype=torch.uint8,
                         device=dev)
        out = torch.empty((B, Hq, 128), dtype=torch.float32, device=dev)
        lse = torch.empty((B, Hq), dtype=torch.float32, device=dev)
        args = (C.byref(Ld), C.byref(c.struct()), Hq, C.c_void_p(q.data_ptr()), float(SCALE),
                C.c_void_p(out.data_ptr()), C.c_void_p(lse.data_ptr()), 0, C.c_void_p(ws.data_ptr()), ws.numel(), sptr)
        for _ in range(3):
            lib.diffkv_decode_attention(*args)
        ev = [(HipEvent(), HipEvent()) for _ in range(reps)]
        rc = 0
        for e in ev:
            flush()
            e[0].record()
            rc |= lib.diffkv_decode_attention(*args)
            e[1].record()
        torch.cuda.synchronize()
        if rc or int(c.status.item()) != 0:
            raise RuntimeError("precision bench failed (%s)" % name)
        us = np.array([a.elapsed_time(b) * 1e3 for a, b in ev])
        kb, vb = kw["k_bits"][sec], kw["v_bits"][sec]
        per_tok = (kb + vb) * 16 + 32          # codes + fp16 scale/zero of K and V
        nbytes = ntok * per_tok + 4 * B * Hkv * (-(-L // Tp)) + B * Hq * 128 * 6
        res["levels"][name] = {"bytes_per_token": per_tok, "us": pct(us),
                               "gbps": nbytes / (us.mean() * 1e-6) / 1e9,
                               "kv_bytes_vs_fp16": per_tok / 512.0}
        log("  precision %-8s %3d B/token: %.1f us, %.0f GB/s" % (name, per_tok, us.mean(), nbytes / us.mean() / 1e3))
        del c, ws
        torch.cuda.empty_cache()
    base = res["levels"]["K8V8"]
    for name, r in res["levels"].items():
        r["speedup_vs_K8V8"] = base["us"]["mean"] / r["us"]["mean"]
        r["bytes_ratio_vs_K8V8"] = base["bytes_per_token"] / r["bytes_per_token"]
    return res


def serving_step(torch, dk, lib, dev, sptr, args):
    """The llama8b shape on `layers` layers sharing one page pool, one step = request
    r = step mod 64 finishes (its pages in every layer recycled by one compaction call),
    a replacement request is prefilled into slot r of every layer while the other 63
    append their newest token (one append call for all layers and requests, as the
    paper runs its KV compaction once per inference step for all requests and layers),
    then attention per layer.  Wall clock around back-to-back steps; HIP events around
    each step's attention calls."""
    from paper_2412_03131_amd import inputs
    t0 = time.time()
    w = inputs.prefill("llama8b")
    B, Hq, Hkv = w["B"], w["Hq"], w["Hkv"]
    NL = args.layers
    nl = w["new_len"].astype(np.int64)
    off = np.concatenate([[0], np.cumsum(nl)])
    K, Wm = args.serving_steps, 16
    steps_total = Wm + 2 * K  # warm-up, the timed pass (no events), the pass with events
    init_hi = w["quota"][:, :, 0].astype(np.int64)
    init_lo = w["quota"][:, :, 1].astype(np.int64)
    L = dk.layout(max_seq_len=int(nl.max()) + steps_total + 16)
    per_table = (-(-(init_hi + steps_total) // 16)) + (-(-init_lo // 32)) + 2
    num_pages = int(NL * per_table.sum() * 1.05) + 1024
    cache = dk.Cache(L, num_pages, NL * B, Hkv, device=dev)
    views = [cache.view(l * B, (l + 1) * B) for l in range(NL)]
    T = lambda a: to_dev(torch, dev, a)
    k_all, v_all, s_all = T(w["k"]), T(w["v"]), T(w["score"])
    quota_all, nl_all = T(w["quota"]), T(w["new_len"])
    ws_a = torch.empty(dk.workspace_size(dk.OP_APPEND, L, B, 0, Hkv, int(nl.sum()) + B) + 256,
                       dtype=torch.uint8, device=dev)
    for v in views:
        dk.quantize_append(v, nl_all, k_all, v_all, s_all, quota=quota_all, total_new=int(nl.sum()),
                           max_new=int(nl.max()), ws=ws_a)
    torch.cuda.synchronize()
    if int(cache.status.item()) != 0:
        raise RuntimeError("serving prefill raised status %d" % int(cache.status.item()))
    steps_in = []
    for s in range(steps_total):
        r = s % B
        d = inputs.decode_token("llama8b", s, B, Hq, Hkv, w["outliers"])
        dk_, dv_, ds_ = T(d["k"]), T(d["v"]), T(d["score"])
        k_s = torch.cat([dk_[:r], k_all[off[r]:off[r + 1]], dk_[r + 1:]])
        v_s = torch.cat([dv_[:r], v_all[off[r]:off[r + 1]], dv_[r + 1:]])
        s_s = torch.cat([ds_[:r], s_all[off[r]:off[r + 1]], ds_[r + 1:]])
        q_np = d["quota"].copy()
        q_np[r] = w["quota"][r]
        n_np = np.ones(B, np.int32)
        n_np[r] = nl[r]
        steps_in.append(dict(r=r, k=torch.cat([k_s] * NL), v=torch.cat([v_s] * NL),
                             score=torch.cat([s_s] * NL), quota=T(np.tile(q_np, (NL, 1, 1))),
                             new_len=T(np.tile(n_np, NL)), total=NL * int(n_np.sum()),
                             maxn=int(n_np.max()), q=T(d["q"])))
    P = L.p_max
    masks = []
    for r in range(B):
        m = torch.zeros((NL * B * Hkv, P), dtype=torch.uint8, device=dev)
        for l in range(NL):
            m[(l * B + r) * Hkv:(l * B + r + 1) * Hkv] = 1
        masks.append(m)
    ws_att = torch.empty(max(256, dk.workspace_size(dk.OP_ATTENTION, L, B, Hq, Hkv, 0, 0)),
                         dtype=torch.uint8, device=dev)
    ws_c = torch.empty(dk.workspace_size(dk.OP_COMPACT, L, NL * B, 0, Hkv), dtype=torch.uint8, device=dev)
    ws_all = torch.empty(dk.workspace_size(dk.OP_APPEND, L, NL * B, 0, Hkv,
                                           max(si["total"] for si in steps_in)) + 256,
                         dtype=torch.uint8, device=dev)
    out = torch.empty((B, Hq, 128), dtype=torch.float32, device=dev)
    lse = torch.empty((B, Hq), dtype=torch.float32, device=dev)
    Lp = C.byref(L)
    cstructs = [v.struct() for v in views]
    call_struct = cache.struct()
    vp = lambda x: C.c_void_p(x.data_ptr())
    attn_args, app_args = [], []
    for si in steps_in:
        app_args.append((Lp, C.byref(call_struct), si["total"], si["maxn"], vp(si["new_len"]),
                         vp(si["k"]), vp(si["v"]), vp(si["score"]), vp(si["quota"]), 0.0, 0.0, 0,
                         vp(ws_all), ws_all.numel(), sptr))
        attn_args.append([(Lp, C.byref(cs), Hq, vp(si["q"]), float(SCALE), vp(out), vp(lse), 0,
                           vp(ws_att), ws_att.numel(), sptr) for cs in cstructs])
    comp_args = [(Lp, C.byref(call_struct), NL * B * Hkv, vp(m), vp(ws_c), ws_c.numel(), sptr)
                 for m in masks]
    seq_rows = [torch.arange(r, NL * B, B, device=dev) for r in range(B)]
    ev = [[HipEvent() for _ in range(4)] for _ in range(K)]

    def run_step(s, e=None):
        si = steps_in[s]
        r = si["r"]
        if e is not None:
            e[0].record()
        rc = lib.diffkv_compact_free_list(*comp_args[r])
        cache.seq_len.index_fill_(0, seq_rows[r], 0)
        if e is not None:
            e[1].record()
        rc |= lib.diffkv_quantize_append(*app_args[s])
        if e is not None:
            e[2].record()
        for l in range(NL):
            rc |= lib.diffkv_decode_attention(*attn_args[s][l])
        if e is not None:
            e[3].record()
        if rc:
            raise RuntimeError("library call failed at serving step %d (rc %d)" % (s, rc))

    len_hi, len_lo = init_hi.copy(), init_lo.copy()
    step_bytes, step_tokens = [], []
    for s in range(steps_total):
        r = s % B
        len_hi += 1
        len_hi[r] = init_hi[r]
        len_lo[r] = init_lo[r]
        step_bytes.append(attn_bytes(len_hi, len_lo, B, Hq, Hkv))
        step_tokens.append(int(len_hi.sum() + len_lo.sum()))
    for s in range(Wm):
        run_step(s)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    for i in range(K):
        run_step(Wm + i)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t1
    for i in range(K):  # per-call times (events between back-to-back calls add gaps)
        run_step(Wm + K + i, ev[i])
    torch.cuda.synchronize()
    status = int(cache.status.item())
    got = cache.len.view(NL, B, Hkv, 2).cpu().numpy()
    if status != 0 or not all(np.array_equal(g[..., 0], len_hi) and np.array_equal(g[..., 1], len_lo)
                              for g in got):
        raise RuntimeError("serving state check failed (status %d)" % status)
    comp_us = np.array([e[0].elapsed_time(e[1]) * 1e3 for e in ev])
    app_us = np.array([e[1].elapsed_time(e[2]) * 1e3 for e in ev])
    att_us = np.array([e[2].elapsed_time(e[3]) * 1e3 / NL for e in ev])
    tok = np.array(step_tokens[Wm:Wm + K], np.float64) * NL
    byt = np.array(step_bytes[Wm + K:], np.float64)
    res = {
        "workload": "llama8b serving step: B=64, Hq=32, Hkv=8, context U[1024,4096], %d layers on one "
                    "pool; per step one request recycled (one compaction call for all layers) and "
                    "re-prefilled while 63 decode (one append call for all layers), then attention "
                    "per layer; built in %.1f s" % (NL, time.time() - t0),
        "kv_tokens_per_s": float(tok.sum() / wall),
        "ms_per_step": wall / K * 1e3,
        "compaction_us": pct(comp_us),
        "append_us": pct(app_us),
        "attention_us_per_launch": pct(att_us),
        "attention_gbps": float(byt.sum() / (att_us.sum() * 1e-6) / 1e9),
        "memory_management_share": float((comp_us + app_us).sum() / (comp_us + app_us + NL * att_us).sum()),
    }
    log("serving step: %.3f ms/step, compaction %.1f us, append %.1f us, attention %.1f us/launch"
        % (res["ms_per_step"], comp_us.mean(), app_us.mean(), att_us.mean()))
    del cache, views, steps_in, masks
    return res


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) > 1:
        print("bench.py runs on one GPU only: the DiffKV path shards by KV head or by request "
              "with no exchange between GPUs, so a multi-GPU figure is N independent copies "
              "of this one.", file=sys.stderr)
        sys.exit(2)
    import torch

    from paper_2412_03131_amd import diffkv as dk

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if args.only == "copy":
        x = torch.empty(1 << 30, dtype=torch.uint8, device=dev)
        y = torch.empty_like(x)
        for _ in range(args.steps):
            y.copy_(x)
        torch.cuda.synchronize()
        log("copied %d x 1 GiB" % args.steps)
        return
    lib = dk.lib()
    stream = torch.cuda.current_stream()
    sptr = C.c_void_p(stream.cuda_stream)
    HipEvent.setup(sptr)
    if args.only == "generation":
        generation_bench(torch, dk, lib, dev, sptr, args.generation_steps)
        return
    if args.only == "prompt":
        prompt_significance_bench(torch, dk, lib, dev, sptr)
        return
    if args.only == "compaction":
        compaction_bench(torch, dk, lib, dev, sptr, args.compaction_rounds)
        return
    flush = Flush(torch, dev)
    wl = build_decode(torch, dk, dev, args.config, min(args.warmup, 8) + 3 * args.steps + 8)
    if args.only == "attention":
        B, Hq, Hkv = wl["w"]["B"], wl["w"]["Hq"], wl["w"]["Hkv"]
        ws = torch.empty(max(256, dk.workspace_size(dk.OP_ATTENTION, wl["L"], B, Hq, Hkv, 0, args.splits)),
                         dtype=torch.uint8, device=dev)
        q = wl["steps"][0]["q"]
        for _ in range(args.warmup + args.steps):
            dk.decode_attention(wl["cache"], q, SCALE, num_splits=args.splits, ws=ws)
        torch.cuda.synchronize()
        log("attention only: %d calls" % (args.warmup + args.steps))
        return
    head = decode_headline(torch, dk, lib, dev, sptr, wl, args, flush)
    extras = {}
    if args.extras == "all":
        extras["significance"] = significance_bench(torch, dk, lib, dev, sptr, wl, flush)
        extras["precisions"] = precision_bench(torch, dk, lib, dev, sptr, flush)
        extras["prompt_significance"] = prompt_significance_bench(torch, dk, lib, dev, sptr)
        if args.config != "llama70b":
            del wl
            torch.cuda.empty_cache()
            wl70 = build_decode(torch, dk, dev, "llama70b", 1)
        else:
            wl70 = wl
        extras["llama70b"] = dict(workload=WORKLOADS["llama70b"].split(";")[0] + "; attention only, "
                                  "flushed before every call; the automatic mode takes one workgroup "
                                  "per table here (256 tables = the resident workgroups of GQA 8)",
                                  **attention_modes(torch, dk, lib, dev, sptr, wl70, args.reps, flush))
        del wl70
        torch.cuda.empty_cache()
        extras["serving_step"] = serving_step(torch, dk, lib, dev, sptr, args)
        torch.cuda.empty_cache()
        extras["compaction"] = compaction_bench(torch, dk, lib, dev, sptr, args.compaction_rounds)
        extras["generation_step"] = generation_bench(torch, dk, lib, dev, sptr, args.generation_steps)
        extras["memory_management"] = memory_management_bench(torch, dk, lib, dev, sptr)
    cpu = None if args.no_cpu_baseline else cpu_baseline(args.config, args.cpu_seconds)
    if cpu is not None and "compaction" in extras:
        c = extras["compaction"]
        c["cpu_oracle_us_per_round"] = cpu["compaction"]["us_per_round"]
        c["gpu_speedup_vs_cpu_oracle"] = cpu["compaction"]["us_per_round"] / c["us_per_round"]
    line = {
        "metric": METRIC,
        "value": head["value"],
        "unit": "KV tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": head["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f16*code->f32",
        "dtype_detail": DTYPE_DETAIL,
        "data": "synthetic",
        "config": {"workload": WORKLOADS[args.config], "global_batch": int(wl_B(args.config)),
                   "attention_splits": args.splits},
        "roofline": {
            "kernel": "diffkv_decode_attention (attn_decode; split tables merged in the same launch)",
            "bound": "hbm",
            "achieved": head["achieved"],
            "peak": HBM_PEAK_GBPS,
            "unit": "GB/s",
            "frac": head["achieved"] / HBM_PEAK_GBPS,
            "traffic": measured_traffic(args.config),
            "bytes_per_launch": head["bytes_per_launch"],
            "us_per_launch": head["us_per_launch"],
            "timing": "HIP events (no system-scope fences) on the launch stream around each step's "
                      "attention call, Infinity "
                      "Cache and L2 evicted before every step (outside the events); mean over K "
                      "steps run right after the back-to-back timed steps, which carry no events",
        },
        "attention": head["attention"],
        "append": head["append"],
        "step": head["step"],
    }
    line.update(extras)
    line["cpu_baseline"] = cpu
    print(json.dumps(line), flush=True)


def wl_B(config):
    from paper_2412_03131_amd import inputs
    return inputs.CONFIGS[config]["B"]


def compaction_bench(torch, dk, lib, dev, sptr, rounds):
    """2^20-page pool, 4096 tables (60% of pages held), Bernoulli(0.35) release per held
    page, then a refill of what each table lost; compaction and refill timed apart."""
    from paper_2412_03131_amd import inputs
    cfg = inputs.CONFIGS["compact"]
    ring, demand = inputs.compaction_setup()
    n_tab, npg = cfg["tables"], cfg["num_pages"]
    L = dk.layout(max_seq_len=(cfg["p_max"] - 1) * 16)
    c = dk.Cache(L, npg, n_tab, 1, device=dev, ring=torch.from_numpy(ring), with_pool=False)
    tpp = torch.tensor([16, 32], dtype=torch.int32, device=dev)
    dk.alloc_pages(c, torch.from_numpy(demand).to(dev))
    c.len.copy_(c.pages * tpp)
    masks = [torch.from_numpy(inputs.release_mask(cfg["seed"], r, n_tab, L.p_max)).to(dev)
             for r in range(rounds)]
    ws_c = torch.empty(dk.workspace_size(dk.OP_COMPACT, L, n_tab, 0, 1), dtype=torch.uint8, device=dev)
    ws_a = torch.empty(dk.workspace_size(dk.OP_ALLOC, L, n_tab, 0, 1), dtype=torch.uint8, device=dev)
    cs = c.struct()
    Lp = C.byref(L)
    live = int(demand.sum())
    ev = [[HipEvent() for _ in range(3)] for _ in range(rounds)]
    before = torch.empty_like(c.pages)
    lost = torch.empty_like(c.pages)
    torch.cuda.synchronize()
    # keep the GPU busy while the host enqueues every round, so the events time
    # the kernels rather than the Python loop
    torch.cuda._sleep(int(2.4e9 * 3e-4 * rounds) + 1)
    for r in range(rounds):
        before.copy_(c.pages)
        ev[r][0].record()
        rc = lib.diffkv_compact_free_list(Lp, C.byref(cs), n_tab, C.c_void_p(masks[r].data_ptr()),
                                          C.c_void_p(ws_c.data_ptr()), ws_c.numel(), sptr)
        ev[r][1].record()
        torch.sub(before, c.pages, out=lost)
        rc |= lib.diffkv_alloc_pages(Lp, C.byref(cs), n_tab, C.c_void_p(lost.data_ptr()),
                                     C.c_void_p(ws_a.data_ptr()), ws_a.numel(), sptr)
        ev[r][2].record()
        torch.mul(c.pages, tpp, out=c.len)
        if rc:
            raise RuntimeError("compaction bench call failed")
    torch.cuda.synchronize()
    ring_ptr = c.ring_ptr.cpu().numpy()
    released = int(ring_ptr[1]) - npg
    if int(c.status.item()) != 0 or int(c.pages.sum().item()) != live:
        raise RuntimeError("compaction bench state check failed")
    cms = np.array([e[0].elapsed_time(e[1]) for e in ev])
    ams = np.array([e[1].elapsed_time(e[2]) for e in ev])
    res = {
        "workload": "2^20 pages, 4096 tables, %d held (60%%), Bernoulli(0.35) release, %d rounds"
                    % (live, rounds),
        "pages_per_s": live / (cms.mean() / 1e3),
        "released_pages_per_s": released / rounds / (cms.mean() / 1e3),
        "us_per_round": float(cms.mean() * 1e3),
        "us_p10_p90": [float(np.percentile(cms, 10) * 1e3), float(np.percentile(cms, 90) * 1e3)],
        "us_median": float(np.median(cms) * 1e3),
        "refill_us_per_round": float(ams.mean() * 1e3),
        "released_per_round": released / rounds,
        "ring_wraps": int(ring_ptr[1] // npg),
    }
    log("compaction: %.1f us/round, %.3g pages/s, refill %.1f us" %
        (res["us_per_round"], res["pages_per_s"], res["refill_us_per_round"]))
    return res


def memory_management_bench(torch, dk, lib, dev, sptr, batches=(8, 32, 128), steps=10, layers=32,
                            threads=None):
    """Memory management per inference step at context 1024 across batch sizes, on the
    GPU and on a multi-threaded host manager (baselines/cpu_manager.c), the comparison
    the paper draws between its on-GPU compaction and on-CPU memory management.  The
    Llama-3-8B shape: 32 layers x 8 KV heads = 256 tables per request, pages from the
    llama8b fractions at 1024 tokens.  Each step one request finishes (its tables in
    every layer released, then refilled by its replacement's prompt pages) and a
    sixteenth of the other tables take one page of decode growth: one compaction plus
    one allocation call for all tables.  Both sides run the same steps from the same
    state and must end bit-identical."""
    from baselines import cpu_manager as cm
    from paper_2412_03131_amd import inputs
    threads = threads or max(1, min(16, cpu_info()[2]))
    res = {"workload": "context 1024, %d layers x 8 KV heads per request, llama8b fractions; per "
                       "step one request recycled and refilled, 1/16 of the other tables grow a "
                       "page; compaction + allocation for all tables" % layers,
           "cpu_threads": threads, "batches": {}}
    for B in batches:
        rng = np.random.default_rng(5 + B)
        H = 8 * layers
        T = B * H
        f_hi = rng.uniform(0.1, 0.5, T)
        f_pr = rng.uniform(0.2, 0.6, T)
        f_pr = np.where(f_hi + f_pr > 1.0, 1.0 - f_hi, f_pr)
        nh = np.floor(f_hi * 1024).astype(np.int64)
        nlo = 1024 - nh - np.floor(f_pr * 1024).astype(np.int64)
        demand0 = np.stack([-(-nh // 16), -(-nlo // 32)], axis=1).astype(np.int32)
        L = dk.layout(max_seq_len=1024 + 16 * (steps + 2))
        num_pages = int(demand0.sum() * 1.25) + 4096
        ring = np.random.default_rng(B).permutation(num_pages).astype(np.int32)
        c = dk.Cache(L, num_pages, B, H, device=dev, ring=torch.from_numpy(ring), with_pool=False)
        dk.alloc_pages(c, torch.from_numpy(demand0).to(dev))
        lens0 = np.stack([nh, nlo], axis=1).astype(np.int32)
        c.len.copy_(torch.from_numpy(lens0).to(dev))
        torch.cuda.synchronize()
        m = cm.Manager(c.page_table.cpu().numpy(), c.pages.cpu().numpy(), lens0, ring,
                       c.ring_ptr.cpu().numpy(), (16, 32), threads)
        rel_np, dem_np = [], []
        for s in range(steps):
            r = s % B
            rel = np.zeros((T, L.p_max), np.uint8)
            rel[r * H:(r + 1) * H] = 1
            dem = np.zeros((T, 2), np.int32)
            dem[(np.arange(T) + s) % 16 == 0, 0] = 1
            dem[r * H:(r + 1) * H] = demand0[r * H:(r + 1) * H]
            rel_np.append(rel)
            dem_np.append(dem)
        rel_d = [torch.from_numpy(x).to(dev) for x in rel_np]
        dem_d = [torch.from_numpy(x).to(dev) for x in dem_np]
        ws_c = torch.empty(dk.workspace_size(dk.OP_COMPACT, L, B, 0, H), dtype=torch.uint8, device=dev)
        ws_a = torch.empty(dk.workspace_size(dk.OP_ALLOC, L, B, 0, H), dtype=torch.uint8, device=dev)
        cs = c.struct()
        Lp = C.byref(L)
        ev = [(HipEvent(), HipEvent()) for _ in range(steps)]
        torch.cuda.synchronize()
        torch.cuda._sleep(int(2.4e9 * 1e-4 * steps) + 1)   # the host enqueues ahead of the GPU
        rc = 0
        for s in range(steps):
            ev[s][0].record()
            rc |= lib.diffkv_compact_free_list(Lp, C.byref(cs), T, C.c_void_p(rel_d[s].data_ptr()),
                                               C.c_void_p(ws_c.data_ptr()), ws_c.numel(), sptr)
            rc |= lib.diffkv_alloc_pages(Lp, C.byref(cs), T, C.c_void_p(dem_d[s].data_ptr()),
                                         C.c_void_p(ws_a.data_ptr()), ws_a.numel(), sptr)
            ev[s][1].record()
        torch.cuda.synchronize()
        if rc or int(c.status.item()) != 0:
            raise RuntimeError("memory management bench: GPU call failed")
        gpu_us = np.array([a.elapsed_time(b) * 1e3 for a, b in ev])
        cpu_us = []
        for s in range(steps):
            t0 = time.perf_counter()
            m.compact(rel_np[s])
            if m.alloc(dem_np[s]):
                raise RuntimeError("memory management bench: host manager refused")
            cpu_us.append((time.perf_counter() - t0) * 1e6)
        m.close()
        same = (np.array_equal(c.page_table.cpu().numpy(), m.table) and np.array_equal(c.ring.cpu().numpy(), m.ring)
                and np.array_equal(c.ring_ptr.cpu().numpy(), m.ring_ptr) and np.array_equal(c.len.cpu().numpy(), m.len))
        if not same:
            raise RuntimeError("memory management bench: GPU and host manager states differ")
        cpu_us = np.array(cpu_us)
        res["batches"][str(B)] = {"tables": T, "live_pages": int(demand0.sum()),
                                  "gpu_us": pct(gpu_us), "cpu_manager_us": pct(cpu_us),
                                  "cpu_over_gpu": float(np.median(cpu_us) / np.median(gpu_us))}
        log("memory management B=%d (%d tables): GPU %.1f us, host manager (%d threads) %.1f us per step"
            % (B, T, np.median(gpu_us), threads, np.median(cpu_us)))
        del c, rel_d, dem_d
    return res


def generation_bench(torch, dk, lib, dev, sptr, steps, window=64):
    """The generation-phase policy (Algorithm 1) on the llama8b workload, one layer:
    prompt phase with the 64-token recent window, then `steps` decode steps of one
    appended token per sequence (score uniform in [0, 2/N), the scale of the prompt's
    normalized scores) followed by one diffkv_generation_step, which HIP events on the
    launch stream time (decide, allocation and apply kernels together)."""
    from paper_2412_03131_amd import inputs
    w = inputs.prefill("llama8b")
    B, Hq, Hkv = w["B"], w["Hq"], w["Hkv"]
    nl = w["new_len"].astype(np.int64)
    L = dk.layout(max_seq_len=int(nl.max()) + steps + 16)
    qh = w["quota"][:, :, 0].astype(np.int64)
    ql = w["quota"][:, :, 1].astype(np.int64)
    npg = int(((-(-(qh + window + steps) // 16)) + (-(-(ql + steps) // 32)) + 2).sum()) + 1024
    c = dk.Cache(L, npg, B, Hkv, device=dev)

    def T(a):
        a = np.ascontiguousarray(a)
        return torch.from_numpy(a.view(np.int16) if a.dtype == np.uint16 else a).to(dev)

    dk.quantize_append(c, T(w["new_len"]), T(w["k"]), T(w["v"]), T(w["score"]), quota=T(w["quota"]),
                       window=window, total_new=int(nl.sum()), max_new=int(nl.max()))
    ws_a = torch.empty(dk.workspace_size(dk.OP_APPEND, L, B, 0, Hkv, B), dtype=torch.uint8, device=dev)
    ws_g = torch.empty(dk.workspace_size(dk.OP_GENERATION, L, B, 0, Hkv), dtype=torch.uint8, device=dev)
    cs = c.struct()
    Lp = C.byref(L)
    vp = lambda x: C.c_void_p(x.data_ptr())
    keep, app = [], []
    ones = T(np.ones(B, np.int32))
    for s in range(steps):
        d = inputs.decode_token("llama8b", s, B, Hq, Hkv, w["outliers"])
        n = (nl + s + 1).astype(np.float32)
        score = (d["score"] * (np.float32(2.0) / n)[:, None]).astype(np.float32)
        t = [T(d["k"]), T(d["v"]), T(score), T(d["quota"])]
        keep.append(t)
        app.append((Lp, C.byref(cs), B, 1, vp(ones), vp(t[0]), vp(t[1]), vp(t[2]), vp(t[3]),
                    0.0, 0.0, window, vp(ws_a), ws_a.numel(), sptr))
    gen = (Lp, C.byref(cs), C.c_float(1.0), C.c_float(0.5), window, vp(ws_g), ws_g.numel(), sptr)
    ev = [(HipEvent(), HipEvent())
          for _ in range(steps)]
    torch.cuda.synchronize()
    lens0, pages0 = c.len.cpu().numpy().copy(), c.pages.cpu().numpy().copy()
    torch.cuda._sleep(int(2.4e9 * 1e-4 * steps) + 1)  # the host enqueues ahead of the GPU
    rc = 0
    for s in range(steps):
        rc |= lib.diffkv_quantize_append(*app[s])
        ev[s][0].record()
        rc |= lib.diffkv_generation_step(*gen)
        ev[s][1].record()
    torch.cuda.synchronize()
    if rc or int(c.status.item()) != 0:
        raise RuntimeError("generation bench failed (rc %d, status %d)" % (rc, int(c.status.item())))
    ms = np.array([a.elapsed_time(b) for a, b in ev])
    lens, pages = c.len.cpu().numpy(), c.pages.cpu().numpy()
    # algorithmic bytes of one call: the decision reads every kept token's position
    # and score (8 B) and every used page-table entry (4 B) plus 40 B of per-table
    # words; applying reads and writes the 1 KiB V code rows of the three pages a
    # table touches (6 KiB) and the codes, metadata, score and position of the two
    # high tokens it reads and the slots it writes (about 0.4 KiB)
    tok = (int(lens0.sum()) + int(lens.sum())) / 2.0
    pg = (int(pages0.sum()) + int(pages.sum())) / 2.0
    nbytes = 8 * tok + 4 * pg + 40 * B * Hkv + (6 * 1024 + 400) * B * Hkv
    res = {
        "workload": "llama8b, 1 layer: B=64, Hkv=8 (512 tables), window 64, alpha_h 1.0, "
                    "alpha_l 0.5, %d decode steps" % steps,
        "us_per_call": float(ms.mean() * 1e3),
        "us_p10_p90": [float(np.percentile(ms, 10) * 1e3), float(np.percentile(ms, 90) * 1e3)],
        "tables_per_s": B * Hkv / (ms.mean() / 1e3),
        "kv_tokens_per_call": tok,
        "algorithmic_bytes_per_call": nbytes,
        "achieved_gbps": nbytes / (ms.mean() / 1e3) / 1e9,
        "bound": "latency: each of the two kernels waits on two dependent rounds of loads",
    }
    log("generation step: %.1f us/call (%d tables)" % (res["us_per_call"], B * Hkv))
    return res




def cpu_info():
    model = None
    try:
        with open("/proc/cpuinfo") as fh:
            for ln in fh:
                if ln.startswith("model name"):
                    model = ln.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        avail = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        avail = os.cpu_count() or 1
    return model, os.cpu_count(), avail


def cpu_baseline(config, seconds):
    """The oracle's fp64 attention on the host, over the first requests of the headline
    workload, each request in its own oracle cache: one thread on request 0, then one
    thread per request on up to 16 requests at once (the machine's CPU share), each looping
    attention passes until `seconds` have passed.  The oracle's C code runs outside the
    interpreter lock, so the threads run in parallel.  Then the serial compaction."""
    import threading

    from oracle import oracle as orc
    from paper_2412_03131_amd import inputs
    model, ncpu, avail = cpu_info()
    nthreads = max(1, min(16, avail, inputs.CONFIGS[config]["B"]))
    t0 = time.time()
    w = inputs.prefill(config, B=nthreads)
    Hkv = w["Hkv"]
    nl = w["new_len"].astype(np.int64)
    off = np.concatenate([[0], np.cumsum(nl)])
    caches = [None] * nthreads

    def build(r):
        Lo = orc.layout(max_seq_len=int(nl[r]) + 16)
        npg = Hkv * (int(nl[r]) // 16 + 4)
        c = orc.Cache(Lo, npg, 1, Hkv)
        orc.quantize_append(c, w["new_len"][r:r + 1], w["k"][off[r]:off[r + 1]], w["v"][off[r]:off[r + 1]],
                            w["score"][off[r]:off[r + 1]], quota=w["quota"][r:r + 1])
        caches[r] = c

    th = [threading.Thread(target=build, args=(r,)) for r in range(nthreads)]
    for x in th:
        x.start()
    for x in th:
        x.join()
    q = [w["q"][r:r + 1] for r in range(nthreads)]
    toks = [int(c.len.sum()) for c in caches]
    log("cpu baseline: %d oracle caches built in %.1f s" % (nthreads, time.time() - t0))

    def passes(r, until, res):
        n = 0
        while True:
            orc.attention(caches[r], q[r], SCALE)
            n += 1
            if time.perf_counter() >= until:
                break
        res[r] = n

    # one thread
    res1 = {}
    t1 = time.perf_counter()
    passes(0, t1 + seconds, res1)
    el1 = time.perf_counter() - t1
    one = toks[0] * res1[0] / el1
    # every thread
    resn = {}
    t2 = time.perf_counter()
    th = [threading.Thread(target=passes, args=(r, t2 + seconds, resn)) for r in range(nthreads)]
    for x in th:
        x.start()
    for x in th:
        x.join()
    el2 = time.perf_counter() - t2
    alln = sum(toks[r] * resn[r] for r in range(nthreads)) / el2
    res = {"value": alln, "unit": "KV tokens/s", "cores": nthreads, "kind": "oracle",
           "sample": "fp64 oracle attention over requests 0-%d of the %s workload (%d KV tokens in all, "
                     "one oracle cache per request), one thread per request, %.1f s wall"
                     % (nthreads - 1, config, sum(toks), el2),
           "single_thread": {"value": one, "cores": 1,
                             "sample": "request 0 (%d KV tokens), %d passes, %.1f s" % (toks[0], res1[0], el1)},
           "cpu_model": model, "nproc": ncpu, "cores_available": avail}
    log("cpu baseline: %.3g KV tokens/s on %d threads, %.3g on one (%s, nproc %s)"
        % (alln, nthreads, one, model, ncpu))
    del caches, w
    res["compaction"] = cpu_compaction(seconds / 4)
    return res


def cpu_compaction(seconds):
    """The oracle's free-list compaction (serial C, one thread) on the compaction
    workload the GPU leg times: 2^20 pages, 4096 tables, Bernoulli(0.35) releases,
    each round followed by the refill, rounds until `seconds` of CPU time."""
    from oracle import oracle as orc
    from paper_2412_03131_amd import inputs
    cfg = inputs.CONFIGS["compact"]
    ring, demand = inputs.compaction_setup()
    n_tab = cfg["tables"]
    Lo = orc.layout(max_seq_len=(cfg["p_max"] - 1) * 16)
    oc = orc.Cache(Lo, cfg["num_pages"], n_tab, 1, ring=ring, with_pool=False)
    orc.alloc_pages(oc, demand)
    tpp = np.array([16, 32])
    oc.len[:] = oc.pages * tpp
    spent, rounds = 0.0, 0
    while spent < seconds:
        rel = inputs.release_mask(cfg["seed"], rounds, n_tab, Lo.p_max)
        before = oc.pages.copy()
        t0 = time.process_time()
        orc.compact(oc, rel)
        spent += time.process_time() - t0
        orc.alloc_pages(oc, (before - oc.pages).astype(np.int32))
        oc.len[:] = oc.pages * tpp
        rounds += 1
    res = {"us_per_round": spent / rounds * 1e6, "rounds": rounds, "cores": 1, "kind": "oracle",
           "sample": "oracle compaction rounds of the 2^20-page, 4096-table workload (refill untimed)"}
    log("cpu compaction: %.0f us/round" % res["us_per_round"])
    return res


if __name__ == "__main__":
    main()
