"""The rule by which the decode kernel composes stability summaries of
consecutive chunks (Algorithm 1's patience counter, split over chunks),
checked on the CPU against the per-block definition.

A chunk's summary, taken with an entering run of 0, is (lead, trail, len,
fis): its leading and trailing stable blocks, its block count, and the first
block where its own run reaches the patience (-1 if none).  Folding an
entering state (stopped, stop step, run) with summaries one chunk at a time
must give the stop that the sequential counter gives over the blocks; and
folding with the composition of several summaries must give the same
integers as folding with them one by one (the kernel composes a window of
64 summaries across the lanes).  The functions below restate the kernel's
fold and composition; the GPU parity tests check the kernel itself."""
from __future__ import annotations

import random

from hypothesis import given, settings
from hypothesis import strategies as st


def summary(bits, p):
    n = len(bits)
    lead = 0
    while lead < n and bits[lead]:
        lead += 1
    trail = 0
    while trail < n and bits[n - 1 - trail]:
        trail += 1
    run, fis = 0, -1
    for i, b in enumerate(bits):
        run = run + 1 if b else 0
        if run >= p:
            fis = i
            break
    return (lead, trail, n, fis)


IDENTITY = (0, 0, 0, -1)


def combine(a, b, p):
    al, at, an, af = a
    bl, bt, bn, bf = b
    lead = an + bl if al == an else al
    trail = bn + at if bt == bn else bt
    if af >= 0:
        fis = af
    elif bl > 0 and at + bl >= p:
        fis = an + (p - at) - 1
    elif bf >= 0:
        fis = an + bf
    else:
        fis = -1
    return (lead, trail, an + bn, fis)


def fold(x, y, t0, p):
    stopped, stop_t, run = x
    if stopped:
        return x
    lead, trail, n, fis = y
    if lead > 0 and run + lead >= p:
        return (1, t0 + (p - run - 1) + 1, run)
    if fis >= 0:
        return (1, t0 + fis + 1, run)
    return (0, 0, run + n if lead == n else trail)


def sequential(bits, p, run0=0):
    """The patience counter over the blocks: (stopped, 1-based stop step)."""
    run = run0
    for t, b in enumerate(bits, start=1):
        run = run + 1 if b else 0
        if run >= p:
            return (1, t)
    return (0, 0)


def chunks_of(bits, sizes):
    out, i = [], 0
    for s in sizes:
        out.append(bits[i:i + s])
        i += s
    return out


@settings(max_examples=400, deadline=None)
@given(st.lists(st.booleans(), min_size=0, max_size=120), st.integers(1, 7),
       st.lists(st.integers(1, 16), min_size=1, max_size=40), st.integers(0, 6))
def test_chunkwise_fold_matches_the_counter(bits, p, sizes, run0):
    run0 = min(run0, p - 1)
    parts = [c for c in chunks_of(bits, sizes) if c]
    x, t0 = (0, 0, run0), 0
    for c in parts:
        x = fold(x, summary(c, p), t0, p)
        t0 += len(c)
    ref = sequential(bits[:t0], p, run0)
    assert (x[0], x[1]) == ref


@settings(max_examples=400, deadline=None)
@given(st.lists(st.booleans(), min_size=0, max_size=200), st.integers(1, 7),
       st.lists(st.integers(1, 16), min_size=1, max_size=64), st.integers(0, 6),
       st.integers(0, 3))
def test_composed_window_folds_like_its_chunks(bits, p, sizes, run0, seed):
    """Composing the summaries in the kernel's tree order (pairs of lanes,
    then pairs of pairs, the earlier chunk on the left) and folding once
    equals folding chunk by chunk."""
    run0 = min(run0, p - 1)
    parts = [c for c in chunks_of(bits, sizes) if c]
    sums = [summary(c, p) for c in parts]
    x1, t0 = (0, 0, run0), 0
    for c, y in zip(parts, sums):
        x1 = fold(x1, y, t0, p)
        t0 += len(c)
    # lanes hold the chunks latest first (lane u: chunk n-1-u), padded with
    # the identity to 64 lanes, reduced with offsets 1, 2, 4, ... 32
    lanes = list(reversed(sums)) + [IDENTITY] * (64 - len(sums))
    d = 1
    while d < 64:
        lanes = [combine(lanes[u + d], lanes[u], p) if u % (2 * d) == 0 and u + d < 64 else lanes[u]
                 for u in range(64)]
        d *= 2
    x2 = fold((0, 0, run0), lanes[0], 0, p)
    if x1[0]:
        assert (x2[0], x2[1]) == (x1[0], x1[1])
    else:
        assert x2 == x1


def test_windows_compose_front_to_back():
    """A long traversal in windows: each window's composition is put in
    front of the later windows' (the kernel walks back), and the fold from
    the start gives the counter's stop."""
    rng = random.Random(7)
    for _ in range(300):
        p = rng.randint(1, 6)
        n_chunks = rng.randint(1, 300)
        parts = [[rng.random() < 0.8 for _ in range(rng.randint(1, 9))] for _ in range(n_chunks)]
        sums = [summary(c, p) for c in parts]
        acc = IDENTITY
        for hi in range(len(sums) - 1, -1, -64):
            window = IDENTITY
            for y in sums[max(0, hi - 63):hi + 1]:
                window = combine(window, y, p)
            acc = combine(window, acc, p)
        bits = [b for c in parts for b in c]
        x = fold((0, 0, 0), acc, 0, p)
        assert (x[0], x[1]) == sequential(bits, p)
