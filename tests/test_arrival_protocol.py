"""Model check of the arrival words (host logic, no GPU).

The attention kernels (split tables merged inside the launch) and the one-token
append (its state written by the last workgroup) find their last arrival with the
routines arrive_count / arrive_takeover / arrive_claim of csrc/common.hpp: a 64-bit
word holding a 44-bit call tag above a 20-bit count, where a word carrying another
call's tag counts as zero.  This file steps a model of those routines, one atomic
operation (load, fetch-add, compare-and-swap) at a time, through random
interleavings of n concurrent arrivals, with and without a concurrent claim, from
stale, garbage and zero words.  Every arrival must obtain a distinct count in
1 .. n (exactly one of them sees n), and the word must end as (tag, n).
"""
import random

CB = 20
MASK = (1 << CB) - 1
M64 = (1 << 64) - 1


class Word:
    def __init__(self, v):
        self.v = v & M64


def takeover(w, old, tag):
    """arrive_takeover: the count before this arrival after its add hit another call's word."""
    old = (old + 1) & M64
    while True:
        cnt = (old & MASK) if (old >> CB) == tag else 0
        nw = (tag << CB) | (cnt + 1)
        yield  # the compare-and-swap, atomic at this step
        if w.v == old:
            w.v = nw
            return cnt
        old = w.v


def arrive_count(w, tag):
    old = w.v
    w.v = (old + 1) & M64
    yield  # the fetch-add
    if (old >> CB) == tag:
        return (old & MASK) + 1
    cnt = yield from takeover(w, old, tag)
    return cnt + 1


def arrive_claim(w, tag):
    old = w.v
    yield  # the load
    while (old >> CB) != tag:
        yield  # the compare-and-swap, atomic at this step
        if w.v == old:
            w.v = tag << CB
            return None
        old = w.v
    return None


def run(word, tag, n, claim, rng):
    w = Word(word)
    gens = [arrive_count(w, tag) for _ in range(n)]
    if claim:
        gens.append(arrive_claim(w, tag))
    res = [None] * len(gens)
    live = list(range(len(gens)))
    while live:
        i = rng.choice(live)
        try:
            next(gens[i])
        except StopIteration as e:
            res[i] = e.value
            live.remove(i)
    return sorted(res[:n]), w.v


def start_word(kind, tag, rng):
    if kind == 0:  # a finished earlier call on the same word
        return (((tag - rng.randint(1, 5)) % (1 << 44)) << CB) | rng.randint(1, 64)
    if kind == 1:  # zero
        return 0
    if kind == 2:  # a count under tag 0 (bytes another kernel left there)
        return rng.randint(1, 4096)
    return rng.randrange(1 << 64)  # anything


def test_arrivals_count_exactly_once_from_any_word():
    rng = random.Random(7)
    trials = 0
    while trials < 20000:
        n = rng.randint(1, 9)
        tag = rng.randrange(1, 1 << 44)
        word = start_word(rng.randrange(4), tag, rng)
        if (word >> CB) == tag or (word & MASK) + n + 1 > MASK:
            continue  # a garbage word equal to this call's tag, or a count carrying into it
        claim = rng.random() < 0.5
        res, final = run(word, tag, n, claim, rng)
        assert res == list(range(1, n + 1)), (word, tag, n, claim, res)
        assert final == (tag << CB) | n, (word, tag, n, claim, final)
        trials += 1


def test_claim_before_arrivals_takes_one_add_each():
    """A claim that completes before any arrival leaves every arrival a single add
    (no compare-and-swap): the path the one-token append takes as a rule."""
    rng = random.Random(8)
    for _ in range(2000):
        n = rng.randint(1, 64)
        tag = rng.randrange(1, 1 << 44)
        word = start_word(rng.randrange(4), tag, rng)
        if (word >> CB) == tag:
            continue
        w = Word(word)
        for _ in arrive_claim(w, tag):
            pass
        assert w.v == tag << CB
        counts = []
        for _ in range(n):
            g = arrive_count(w, tag)
            steps = 0
            try:
                while True:
                    next(g)
                    steps += 1
            except StopIteration as e:
                counts.append(e.value)
            assert steps == 1
        assert counts == list(range(1, n + 1))


def test_the_model_catches_a_dropped_tag_check():
    """A mistaken variant (a stale word's count taken as this call's) fails the check."""
    def bad_count(w, tag):
        old = w.v
        w.v = (old + 1) & M64
        yield
        return (old & MASK) + 1
    w = Word((123 << CB) | 5)
    tag = 456
    gens = [bad_count(w, tag) for _ in range(3)]
    res = []
    for g in gens:
        try:
            while True:
                next(g)
        except StopIteration as e:
            res.append(e.value)
    assert sorted(res) != [1, 2, 3]
