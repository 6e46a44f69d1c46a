"""Pins of the slot-protocol oracle (no GPU).

The state machine of a server step (EaaS §3.2 flags, §3.3 server loop, §3.4
offline clients): hand-worked cases for which slots a step takes, the
invariants every step keeps (slots in other states, and payload rows past a
request, are never written; taken slots end at flag 2), and the results of
taken requests against token-wise brute force with each request's own layer
weights.  Planted mistakes in the slot selection fail these pins.
"""
import numpy as np
import pytest

from oracle import eaas_oracle as O
from oracle import server_oracle as SV
from paper_2509_17863_amd import synth

E, H, I, K = 6, 64, 32, 2


def hand(flags, sizes, caps, total):
    t, c = SV.take_slots(flags, sizes, caps, total)
    return t.tolist(), c.tolist()


def test_take_slots_hand_cases():
    # only flag 1 is taken; 0 (empty), 2 (done), 3 (offline) are left alone
    assert hand([1, 0, 1, 3, 1, 2], [4, 9, 2, 9, 3, 9], [8] * 6, 100) == (
        [True, False, True, False, True, False], [4, 0, 2, 0, 3, 0])
    # batch sizes are clamped to the payload capacity and to >= 0
    assert hand([1, 1, 1], [20, -5, 7], [8, 8, 8], 100) == ([True, True, True], [8, 0, 7])
    # capacity: slot 1 does not fit, so neither it nor anything after it is taken
    assert hand([1, 1, 1, 1], [5, 10, 1, 1], [16] * 4, 12) == ([True, False, False, False],
                                                             [5, 0, 0, 0])
    # an empty ready request is taken (and answered) at no capacity cost
    assert hand([1, 1], [0, 12], [16, 16], 12) == ([True, True], [0, 12])
    assert hand([], [], [], 5) == ([], [])


def _layers(nl, seed):
    out = []
    for L in range(nl):
        d = synth.make_inputs(1, H, I, E, K, seed + 100 * L)
        out.append({key: d[key] for key in ("wdtype", "w_gate_up", "w_down", "w_gate_up_scale",
                                            "w_down_scale")})
    return out


def _slots(specs, seed=3):
    """specs: (flag, layer, n, capacity)."""
    rng = np.random.default_rng(seed)
    slots = []
    for flag, layer, n, cap in specs:
        x = synth.bf16_bits_from_f32(rng.standard_normal((cap, H)).astype(np.float32))
        ids = rng.integers(-1, E + 1, size=(cap, K)).astype(np.int32)
        w = rng.random((cap, K)).astype(np.float32)
        slots.append(dict(flag=flag, layer=layer, n=n, x=x, topk_ids=ids, topk_weights=w))
    return slots


def test_server_step_state_machine_and_results():
    layers = _layers(2, 7)
    specs = [(1, 0, 5, 8), (0, 1, 4, 8), (1, 1, 7, 7), (3, 0, 6, 8), (1, 0, 0, 4), (2, 1, 3, 8),
             (1, 5, 3, 4), (1, 1, 9, 12)]
    slots = _slots(specs)
    flags, xs, res = SV.server_step(slots, layers, E, cap_total=20)
    taken, counts = SV.take_slots([s["flag"] for s in slots], [s["n"] for s in slots],
                                  [s["x"].shape[0] for s in slots], 20)
    # 5 + 7 + 0 + 3 = 15 tokens fit; slot 7 (9 more) does not and stays ready
    assert taken.tolist() == [True, False, True, False, True, False, True, False]
    assert flags.tolist() == [2, 0, 2, 3, 2, 2, 2, 1]
    for b, s in enumerate(slots):
        n = int(counts[b])
        # payload rows past the request, and slots not taken, are untouched
        assert np.array_equal(xs[b][n:], s["x"][n:])
        if not taken[b] or n == 0:
            assert np.array_equal(xs[b], s["x"])
            continue
        if not (0 <= s["layer"] < len(layers)):
            assert np.all(res[b] == 0) and np.all(xs[b][:n] == 0)
            continue
        req = dict(layers[s["layer"]], E=E, H=H, I=I, k=K, T=n, x=s["x"][:n],
                   topk_ids=s["topk_ids"][:n], topk_weights=s["topk_weights"][:n])
        ref = O.brute_force_tokens(req, range(n))
        assert np.abs(res[b] - ref).max() <= 1e-9 * max(1.0, np.abs(ref).max())
        assert np.array_equal(xs[b][:n], O.f32_to_bf16_rne(res[b].astype(np.float32)))


def test_server_step_nothing_ready():
    layers = _layers(1, 8)
    slots = _slots([(0, 0, 3, 4), (3, 0, 2, 4), (2, 0, 1, 4)])
    flags, xs, res = SV.server_step(slots, layers, E, cap_total=16)
    assert flags.tolist() == [0, 3, 2]
    assert all(np.array_equal(a, s["x"]) for a, s in zip(xs, slots))
    assert res == [None, None, None]


# ------------------------------------------------------- planted mistakes
_TAKE = SV.take_slots


def _take_also_empty(flags, sizes, caps, total):
    return _TAKE([1 if f in (0, 1) else f for f in flags], sizes, caps, total)


def _take_skip_not_break(flags, sizes, caps, total):
    taken = np.zeros(len(flags), dtype=bool)
    counts = np.zeros(len(flags), dtype=np.int64)
    t = 0
    for b, f in enumerate(flags):
        n = min(max(int(sizes[b]), 0), int(caps[b]))
        if f == 1 and t + n <= total:
            taken[b], counts[b], t = True, n, t + n
    return taken, counts


@pytest.mark.parametrize("mutant", [_take_also_empty, _take_skip_not_break])
def test_planted_slot_selection_mistakes_fail(mutant, monkeypatch):
    monkeypatch.setattr(SV, "take_slots", mutant)
    with pytest.raises(AssertionError):
        test_take_slots_hand_cases()
