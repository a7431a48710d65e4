"""Seeded synthetic inputs for the DiffKV hot path.

This module only draws random numbers and shapes them; it holds none of the
method's arithmetic (no classing, quantization, allocation or attention).
The same arrays feed the GPU library and the CPU oracle.

Workloads (sizes of the paper's Llama-3-8B, Qwen/QwQ-32B and Llama-3-70B
decode shapes; the paper's datasets are stood in for by these draws):

  tiny      B=2,  Hq=4,  Hkv=4, L=512,            split 40/40/20 (seed 0)
  llama8b   B=64, Hq=32, Hkv=8, L~U{1024..4096},  f_hi~U[.1,.5], f_pr~U[.2,.6] (seed 1)
  long32k   B=16, Hq=40, Hkv=8, L=32768,          f_pr=0.1+0.8*Beta(2,2), kept split
                                                  evenly high/low, then 1-token
                                                  decode steps (seed 2)
  llama70b  B=32, Hq=64, Hkv=8, L=8192,           split 30/40/30 (seed 3)
  compact   2^20-page pool, 4096 tables, 60% allocated, Bernoulli(0.35)
            release per page per round, 100 rounds (seed 4)

Value distributions: q, k, v ~ N(0,1) drawn in fp32 and rounded to fp16;
each KV head has 4 key outlier channels (drawn without replacement) scaled
by 10 before rounding.  Token importance: per (sequence, KV head) a random
permutation pi of the token positions gives score_j = (pi_j+1)^-1.1 / H_L
(Zipf exponent 1.1, distinct, sums to 1), stored fp32.  Counts from
fractions: n_hi = floor(f_hi*L), n_pr = floor(f_pr*L), n_lo = L-n_hi-n_pr.
"""
import numpy as np

HEAD_DIM = 128
ZIPF_S = 1.1
N_OUTLIER = 4
OUTLIER_SCALE = 10.0

CONFIGS = {
    "tiny": dict(B=2, Hq=4, Hkv=4, L=512, seed=0),
    "llama8b": dict(B=64, Hq=32, Hkv=8, L=(1024, 4096), seed=1),
    "long32k": dict(B=16, Hq=40, Hkv=8, L=32768, seed=2, decode_steps=64),
    "llama70b": dict(B=32, Hq=64, Hkv=8, L=8192, seed=3),
    "compact": dict(num_pages=1 << 20, tables=4096, alloc_frac=0.6, release_p=0.35,
                    rounds=100, p_max=256, seed=4),
}


def _streams(seed, n):
    return [np.random.default_rng(s) for s in np.random.SeedSequence(seed).spawn(n)]


def f16_bits(x):
    """fp32 array -> fp16 bit patterns (numpy's round-to-nearest-even cast)."""
    return np.asarray(x, np.float32).astype(np.float16).view(np.uint16)


def zipf_scores(rng, n):
    """Distinct heavy-tailed scores summing to 1, in random position order."""
    r = np.arange(1, n + 1, dtype=np.float64) ** (-ZIPF_S)
    r /= r.sum()
    pi = rng.permutation(n)
    return r[pi].astype(np.float32)


def outlier_channels(rng, Hkv, D=HEAD_DIM):
    return np.stack([rng.choice(D, N_OUTLIER, replace=False) for _ in range(Hkv)])


def draw_kv(rng_k, rng_v, rows, Hkv, outl, D=HEAD_DIM):
    k = rng_k.standard_normal((rows, Hkv, D), dtype=np.float32)
    for h in range(Hkv):
        k[:, h, outl[h]] *= OUTLIER_SCALE
    v = rng_v.standard_normal((rows, Hkv, D), dtype=np.float32)
    return f16_bits(k), f16_bits(v)


def counts_from_fractions(L, f_hi, f_pr):
    n_hi = np.floor(np.asarray(f_hi) * L).astype(np.int64)
    n_pr = np.floor(np.asarray(f_pr) * L).astype(np.int64)
    return n_hi, L - n_hi - n_pr


def prefill(name, seed=None, B=None, L=None):
    """Prompt-phase inputs of a decode workload.

    Returns dict with new_len [B] int32, k/v [rows][Hkv][D] fp16 bits,
    score [rows][Hkv] fp32, quota [B][Hkv][2] int32, q [B][Hq][D] fp16 bits,
    plus the shape numbers.  B and L may be overridden (smaller parity cases).
    """
    cfg = dict(CONFIGS[name])
    seed = cfg["seed"] if seed is None else seed
    B = cfg["B"] if B is None else B
    Hq, Hkv = cfg["Hq"], cfg["Hkv"]
    r_len, r_frac, r_q, r_k, r_v, r_s, r_o = _streams(seed, 7)
    Lc = cfg["L"] if L is None else L
    if isinstance(Lc, tuple):
        new_len = r_len.integers(Lc[0], Lc[1] + 1, size=B).astype(np.int32)
    else:
        new_len = np.full(B, Lc, np.int32)
    quota = np.zeros((B, Hkv, 2), np.int32)
    for b in range(B):
        n = int(new_len[b])
        if name == "tiny":
            nh, nl = counts_from_fractions(n, np.full(Hkv, 0.4), np.full(Hkv, 0.2))
        elif name == "llama8b":
            f_hi = r_frac.uniform(0.1, 0.5, Hkv)
            f_pr = r_frac.uniform(0.2, 0.6, Hkv)
            f_pr = np.where(f_hi + f_pr > 1.0, 1.0 - f_hi, f_pr)
            nh, nl = counts_from_fractions(n, f_hi, f_pr)
        elif name == "long32k":
            f_pr = 0.1 + 0.8 * r_frac.beta(2.0, 2.0, Hkv)
            kept = n - np.floor(f_pr * n).astype(np.int64)
            nh = kept // 2
            nl = kept - nh
        elif name == "llama70b":
            nh, nl = counts_from_fractions(n, np.full(Hkv, 0.3), np.full(Hkv, 0.3))
        else:
            raise ValueError(name)
        quota[b, :, 0] = nh
        quota[b, :, 1] = nl
    rows = int(new_len.sum())
    outl = outlier_channels(r_o, Hkv)
    k, v = draw_kv(r_k, r_v, rows, Hkv, outl)
    score = np.empty((rows, Hkv), np.float32)
    off = 0
    for b in range(B):
        n = int(new_len[b])
        for h in range(Hkv):
            score[off:off + n, h] = zipf_scores(r_s, n)
        off += n
    q = f16_bits(r_q.standard_normal((B, Hq, HEAD_DIM), dtype=np.float32))
    return dict(name=name, B=B, Hq=Hq, Hkv=Hkv, new_len=new_len, k=k, v=v, score=score,
                quota=quota, q=q, outliers=outl, max_len=int(new_len.max()))


def uniform_cache(B, Hq, Hkv, L, seed=5):
    """A decode cache's inputs with no pruning and one precision for every token: the
    llama8b value distributions (q, k, v ~ N(0,1), 4 key outlier channels x10 per KV head),
    L tokens per sequence, Zipf scores.  Returns new_len, k, v, score, q."""
    r_k, r_v, r_s, r_q, r_o = _streams(seed, 5)
    outl = outlier_channels(r_o, Hkv)
    k, v = draw_kv(r_k, r_v, B * L, Hkv, outl)
    score = np.empty((B * L, Hkv), np.float32)
    for b in range(B):
        for h in range(Hkv):
            score[b * L:(b + 1) * L, h] = zipf_scores(r_s, L)
    q = f16_bits(r_q.standard_normal((B, Hq, HEAD_DIM), dtype=np.float32))
    return dict(new_len=np.full(B, L, np.int32), k=k, v=v, score=score, q=q)


def prompt_queries(name, rows, seed=None):
    """Queries of the prompt rows of a workload: fp16 bits [rows][Hq][D], N(0,1)."""
    cfg = CONFIGS[name]
    seed = cfg["seed"] + 17 if seed is None else seed
    (r_q,) = _streams(seed, 1)
    return f16_bits(r_q.standard_normal((rows, cfg["Hq"], HEAD_DIM), dtype=np.float32))


def decode_token(name, step, B, Hq, Hkv, outliers, seed=None):
    """One generated token per sequence: k/v [B][Hkv][D], score [B][Hkv],
    quota (1, 0) per table (the new token enters the recent window), new q."""
    cfg = CONFIGS[name]
    seed = cfg["seed"] if seed is None else seed
    r_q, r_k, r_v, r_s = _streams(seed * 1000003 + 7919 * (step + 1), 4)
    k, v = draw_kv(r_k, r_v, B, Hkv, outliers)
    score = r_s.random((B, Hkv), dtype=np.float32)
    quota = np.zeros((B, Hkv, 2), np.int32)
    quota[:, :, 0] = 1
    q = f16_bits(r_q.standard_normal((B, Hq, HEAD_DIM), dtype=np.float32))
    return dict(new_len=np.ones(B, np.int32), k=k, v=v, score=score, quota=quota, q=q)


def compaction_setup(seed=None, num_pages=None, tables=None, alloc_frac=None):
    """Initial free-list permutation and per-table page counts {high, low}."""
    cfg = CONFIGS["compact"]
    seed = cfg["seed"] if seed is None else seed
    num_pages = cfg["num_pages"] if num_pages is None else num_pages
    tables = cfg["tables"] if tables is None else tables
    alloc_frac = cfg["alloc_frac"] if alloc_frac is None else alloc_frac
    r_ring, r_w, r_u = _streams(seed, 3)
    ring = r_ring.permutation(num_pages).astype(np.int32)
    total = int(np.floor(alloc_frac * num_pages))
    w = r_w.uniform(0.5, 1.5, tables)
    pages = np.floor(total * w / w.sum()).astype(np.int64)
    rem = total - int(pages.sum())
    pages[:rem] += 1
    u = r_u.uniform(0.0, 1.0, tables)
    hi = np.floor(u * pages).astype(np.int64)
    demand = np.stack([hi, pages - hi], axis=1).astype(np.int32)
    return ring, demand


def release_mask(seed, round_idx, tables, p_max, p=None):
    """Bernoulli(p) per table slot; the kernel ignores slots that hold no page."""
    p = CONFIGS["compact"]["release_p"] if p is None else p
    rng = np.random.default_rng(np.random.SeedSequence(seed).spawn(round_idx + 1)[round_idx])
    return (rng.random((tables, p_max)) < p).astype(np.uint8)
