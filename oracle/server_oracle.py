"""CPU oracle for one expert server step over its clients' buffer slots.

TEST INFRASTRUCTURE ONLY.  Imported by ``tests/`` (and through ``oracle``);
nothing in the product library imports, links or runs it, and it shares no
code with the HIP path.

What it models (EaaS §3.2 "Shared Communication Buffer Design", §3.3
"Asynchronous Server Operation", §3.4 "Fault Tolerance"):
  * every client owns one slot on the server: a state flag, a header with the
    layer id and the batch size, and a payload with the hidden states, an
    expert id per token slot and the router scores;
  * flag values: 0 empty (the client may write), 1 client write done (ready
    for the server), 2 server computation done (the client may read),
    3 offline (a client the monitor reported dead: its slot is left alone);
  * one server step takes the slots that are ready when it looks, runs them
    as one dynamic batch, writes each request's weighted sums back into its
    own payload (over the hidden states) and sets those slots' flags to 2.
    Nothing else is written: the server never touches a slot in another
    state and never initiates anything.

Readings where the paper is silent (binding for the library as well):
  * batch capacity: the ready slots are taken in slot order while the running
    token total fits the step's capacity; the first ready slot that does not
    fit, and every ready slot after it, stay at flag 1 for a later step;
  * a request whose layer id names no layer of this server is taken and
    answered with zeros (no expert of it lives here), flag set to 2;
  * batch sizes are clamped to [0, payload capacity]; a batch size of 0 is a
    valid empty request (taken, flag set to 2, nothing else written);
  * a server holding several layers batches requests of different layers
    together: expert e of layer L is group L*E + e of one grouped step.
"""
from __future__ import annotations

import numpy as np

from .eaas_oracle import expert_forward, f32_to_bf16_rne

__all__ = ["EMPTY", "READY", "DONE", "OFFLINE", "take_slots", "server_step"]

EMPTY, READY, DONE, OFFLINE = 0, 1, 2, 3


def take_slots(flags, batch_sizes, capacities, cap_total):
    """Which slots one step takes, and their token counts."""
    taken = np.zeros(len(flags), dtype=bool)
    counts = np.zeros(len(flags), dtype=np.int64)
    total = 0
    for b, f in enumerate(flags):
        if f != READY:
            continue
        n = min(max(int(batch_sizes[b]), 0), int(capacities[b]))
        if total + n > cap_total:
            break
        taken[b] = True
        counts[b] = n
        total += n
    return taken, counts


def server_step(slots, layers, E, cap_total):
    """One step over `slots` (list of dicts: flag, layer, n, x bits [cap,H],
    topk_ids, topk_weights) with per-layer weights `layers` (list of dicts with
    wdtype, w_gate_up, w_down and scales).  Returns (new flags, per slot the
    payload x after the step as bf16 bits, per slot the fp64 results of the
    taken rows or None)."""
    flags = np.array([s["flag"] for s in slots])
    taken, counts = take_slots(flags, [s["n"] for s in slots],
                               [s["x"].shape[0] for s in slots], cap_total)
    new_flags = flags.copy()
    new_flags[taken] = DONE
    xs = [s["x"].copy() for s in slots]
    res = [None] * len(slots)
    for L, lw in enumerate(layers):
        members = [b for b in range(len(slots)) if taken[b] and slots[b]["layer"] == L and counts[b]]
        if not members:
            continue
        H = slots[members[0]]["x"].shape[1]
        k = slots[members[0]]["topk_ids"].shape[1]
        batch = dict(lw, E=E, H=H, I=lw["w_down"].shape[2], k=k,
                     T=int(sum(counts[b] for b in members)),
                     x=np.concatenate([slots[b]["x"][: counts[b]] for b in members]),
                     topk_ids=np.concatenate([slots[b]["topk_ids"][: counts[b]] for b in members]),
                     topk_weights=np.concatenate([slots[b]["topk_weights"][: counts[b]]
                                                  for b in members]))
        out = expert_forward(batch)["out"]
        p = 0
        for b in members:
            n = int(counts[b])
            res[b] = out[p: p + n]
            xs[b][:n] = f32_to_bf16_rne(out[p: p + n].astype(np.float32))
            p += n
    for b in range(len(slots)):
        n = int(counts[b])
        if taken[b] and n and not (0 <= slots[b]["layer"] < len(layers)):
            res[b] = np.zeros((n, slots[b]["x"].shape[1]))
            xs[b][:n] = 0
    return new_flags, xs, res
