"""Pins of the multi-client dynamic-batch oracle (no GPU).

Algorithm 1 (EaaS §4): its literal steps are checked against the closed form
they must reduce to -- a grid-stride walk over the concatenation of the
batches, so global token g = P_b + t is visited exactly once, by block
g mod grid -- on hand-made and random count vectors (empty and negative
counts, grids larger than the batch, a grid of one).
Dynamic batching (§3.3): the step on the aggregated batch, handed back per
request, equals the step run on each request alone (the server is
stateless, so a token's output depends on that token only).
Planted mistakes in Algorithm 1 fail these pins.
"""
import numpy as np
import pytest

from oracle import eaas_oracle as O
from oracle import segments_oracle as S
from paper_2509_17863_amd import synth


def closed_form(num_tokens, grid):
    counts = [max(int(n), 0) for n in num_tokens]
    want = [[] for _ in range(grid)]
    g = 0
    for b, n in enumerate(counts):
        for t in range(n):
            want[(g + t) % grid].append((b, t))
        g += n
    return want


def check_visits(visits, num_tokens, grid):
    assert len(visits) == grid
    assert visits == closed_form(num_tokens, grid)
    flat = [v for blk in visits for v in blk]
    counts = [max(int(n), 0) for n in num_tokens]
    assert sorted(flat) == [(b, t) for b, n in enumerate(counts) for t in range(n)]


CASES = [
    ([5], 2), ([5], 8), ([0], 3), ([3, 0, 4], 2), ([0, 0, 0], 4), ([1, 1, 1, 1], 3),
    ([7, 2, 9, 0, 1], 4), ([2, 3], 1), ([10, -3, 4], 3), ([64, 64], 64), ([65, 63], 64),
]


@pytest.mark.parametrize("num_tokens,grid", CASES)
def test_algorithm1_closed_form(num_tokens, grid):
    check_visits(S.algorithm1_visits(num_tokens, grid), num_tokens, grid)


def test_algorithm1_random():
    rng = np.random.default_rng(5)
    for _ in range(200):
        nb = int(rng.integers(1, 9))
        counts = rng.integers(-2, 40, size=nb)
        counts[rng.random(nb) < 0.3] = 0
        grid = int(rng.integers(1, 50))
        check_visits(S.algorithm1_visits(counts, grid), counts, grid)


def test_algorithm1_single_batch_is_grid_stride():
    v = S.algorithm1_visits([11], 4)
    assert v == [[(0, t) for t in range(b, 11, 4)] for b in range(4)]


def _requests(sizes, H=64, I=32, E=6, k=2, seed=3, wdtype="bf16"):
    T = sum(sizes)
    d = synth.make_inputs(max(T, 1), H, I, E, k, seed)
    reqs, p = [], 0
    for n in sizes:
        r = dict(d)
        # each payload buffer holds more rows than the request uses
        cap = n + 3
        x = np.zeros((cap, H), dtype=d["x"].dtype)
        ids = np.full((cap, k), -1, dtype=np.int32)
        w = np.zeros((cap, k), dtype=np.float32)
        x[:n], ids[:n], w[:n] = d["x"][p:p + n], d["topk_ids"][p:p + n], d["topk_weights"][p:p + n]
        r.update(T=cap, x=x, topk_ids=ids, topk_weights=w, n=n)
        reqs.append(r)
        p += n
    return d, reqs


def test_dynamic_batch_concatenates_in_slot_order():
    d, reqs = _requests([3, 0, 5, 2])
    b = S.dynamic_batch(reqs)
    assert b["T"] == 10
    assert np.array_equal(b["x"], d["x"][:10])
    assert np.array_equal(b["topk_ids"], d["topk_ids"][:10])
    assert np.array_equal(b["topk_weights"], d["topk_weights"][:10])


@pytest.mark.parametrize("sizes", [[4, 0, 7, 1], [9], [0, 0, 3], [1, 1, 1, 1, 1]])
def test_segmented_forward_equals_each_request_alone(sizes):
    d, reqs = _requests(sizes)
    got = S.segmented_forward(reqs)
    for r, g in zip(reqs, got):
        assert g.shape == (r["n"], d["H"])
        if r["n"] == 0:
            continue
        alone = dict(r)
        alone.update(T=r["n"], x=r["x"][: r["n"]], topk_ids=r["topk_ids"][: r["n"]],
                     topk_weights=r["topk_weights"][: r["n"]])
        ref = O.brute_force_tokens(alone, range(r["n"]))
        assert np.abs(g - ref).max() <= 1e-9 * max(1.0, np.abs(ref).max())


def test_segmented_forward_all_empty():
    _, reqs = _requests([0, 0])
    got = S.segmented_forward(reqs)
    assert [g.shape for g in got] == [(0, 64), (0, 64)]


# ------------------------------------------------------- planted mistakes
def _alg1_no_carry(num_tokens, grid):
    # mistake: restart every batch at token blockIdx (drops the carried overshoot)
    counts = [max(int(n), 0) for n in num_tokens]
    out = []
    for block in range(grid):
        mine = []
        for b, n in enumerate(counts):
            t = block
            while t < n:
                mine.append((b, t))
                t += grid
        out.append(mine)
    return out


def _alg1_carry_sign(num_tokens, grid):
    # mistake: carry token_id + n instead of token_id - n
    counts = [max(int(n), 0) for n in num_tokens]
    out = []
    for block in range(grid):
        mine, t = [], block
        for b, n in enumerate(counts):
            while t < n:
                mine.append((b, t))
                t += grid
            t = t - n if b == 0 else t + n
        out.append(mine)
    return out


@pytest.mark.parametrize("mutant", [_alg1_no_carry, _alg1_carry_sign])
def test_planted_algorithm1_mistakes_fail(mutant):
    failed = False
    for num_tokens, grid in CASES:
        try:
            check_visits(mutant(num_tokens, grid), num_tokens, grid)
        except AssertionError:
            failed = True
    assert failed
