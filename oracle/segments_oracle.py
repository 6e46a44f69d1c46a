"""CPU oracle for the multi-client dynamic batch of an expert server step.

TEST INFRASTRUCTURE ONLY.  Imported by ``tests/`` (and through ``oracle``);
nothing in the product library imports, links or runs it, and it shares no
code with the HIP path.

What it computes (EaaS §3.3 "Asynchronous Server Operation"): the server
aggregates the ready requests of several clients into one dynamic batch,
runs the step on it, and writes each client's rows of the weighted sum back
into that client's own payload.  A request is the payload of §3.2 (hidden
states, an expert id per token slot, the router scores) with its header's
batch size; a client whose batch size is 0 contributes nothing.

Algorithm 1 (§4, "Iterate tokens with various length of batches") is how a
static grid walks such a batch: block b starts at token b of the first
batch, strides by the grid size inside a batch, and carries the overshoot
into the next batch (skipping empty ones), with the per-batch token counts
held in shared memory.  ``algorithm1_visits`` runs those steps literally.
"""
from __future__ import annotations

import numpy as np

from .eaas_oracle import expert_forward

__all__ = ["algorithm1_visits", "dynamic_batch", "segmented_forward"]


def algorithm1_visits(num_tokens, grid: int):
    """Algorithm 1 for every block of a grid of `grid` blocks.

    Returns, per block, the list of (batch_id, token_id) pairs on which the
    block calls compute_func, in the order it calls them.  Negative counts
    are treated as empty batches (a count is data written by a client)."""
    counts = [max(int(n), 0) for n in num_tokens]   # the shared-memory copy
    visits = []
    for block in range(grid):
        mine = []
        token_id = block
        for batch_id, n in enumerate(counts):
            while token_id < n:
                mine.append((batch_id, token_id))
                token_id += grid
            token_id -= n
        visits.append(mine)
    return visits


def dynamic_batch(requests) -> dict:
    """Aggregate ready requests (dicts with the payload arrays and "n", the
    header's batch size) into one batch, in slot order: the tokens of request
    0, then those of request 1, ...  Only the first n rows of a payload are
    part of the request."""
    first = requests[0]
    H, I, E, k = first["H"], first["I"], first["E"], first["k"]
    parts = [(r["x"][: r["n"]], r["topk_ids"][: r["n"]], r["topk_weights"][: r["n"]])
             for r in requests]
    batch = dict(first)
    batch.update(
        T=int(sum(r["n"] for r in requests)), H=H, I=I, E=E, k=k,
        x=np.concatenate([p[0] for p in parts]).reshape(-1, H),
        topk_ids=np.concatenate([p[1] for p in parts]).reshape(-1, k),
        topk_weights=np.concatenate([p[2] for p in parts]).reshape(-1, k))
    return batch


def segmented_forward(requests, weights=None):
    """The server step on a dynamic batch: the weighted sums of the whole
    batch, handed back per request (request i gets rows P_i .. P_i + n_i,
    P_i the tokens of the requests before it).  Returns a list of fp64
    [n_i, H] arrays."""
    batch = dynamic_batch(requests)
    out = expert_forward(batch, weights)["out"] if batch["T"] else np.zeros((0, batch["H"]))
    res, p = [], 0
    for r in requests:
        res.append(out[p: p + r["n"]])
        p += r["n"]
    return res
