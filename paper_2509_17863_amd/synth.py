"""Seeded synthetic inputs for one expert server's forward step.

This module is shared by the tests, the benchmark and the CPU oracle's
callers.  It produces the request payload (hidden states, per-token expert
ids and router scores, as carried in a client's buffer slot, §3.2) and the
resident experts' weights.  It holds none of the server's arithmetic: the
router below plays the attention client's role (softmax, top-k, renormalise)
and only decides which ids and scores arrive.

Recipe (five named workloads, seeds 0..4):
  * RNG: numpy PCG64 from SeedSequence(seed), spawned in the fixed order
    [x, w_gate_up, w_down, logits, rank]; the two weight streams are spawned
    again per expert so experts can be generated independently (and in
    parallel threads) with a result that does not depend on thread count.
  * x ~ N(0,1) drawn in fp32, rounded to bf16 (round-to-nearest-even).
  * W_gate_up[E,2I,H] (gate rows [0,I), up rows [I,2I)) and W_down[E,H,I]
    ~ N(0, std=1/sqrt(fan_in)), fan_in = H and I respectively, drawn in fp32
    then rounded to bf16, or quantised to fp8-e4m3fn with one fp32 scale per
    128x128 block, s = amax/448 (s = 1 for an all-zero block).
  * logits ~ N(0,1) in fp64 plus a per-expert bias -alpha*ln(rank_e) for the
    Zipf-skewed workloads (rank = a random permutation of 1..E); p = softmax;
    top-k by descending logit, ties to the lower id; weights p_sel/sum(p_sel)
    as fp32; ids int32.

Arrays: bf16 tensors are uint16 bit patterns, fp8 tensors uint8 bit patterns.
"""
from __future__ import annotations

import hashlib
import os
from concurrent.futures import ThreadPoolExecutor
from dataclasses import dataclass, asdict

import numpy as np

__all__ = ["Workload", "WORKLOADS", "make_inputs", "make_workload", "manifest",
           "bf16_bits_from_f32", "fp8e4m3_quantize_blocks", "route_tokens"]


@dataclass(frozen=True)
class Workload:
    name: str
    T: int
    H: int
    I: int
    E: int
    k: int
    seed: int
    zipf: float | None = None     # alpha of the per-expert logit bias, None = no bias
    wdtype: str = "bf16"          # "bf16" or "fp8"
    act8: bool = False            # fp8 activations too (fp8 weights only)

    @property
    def R(self) -> int:
        return self.T * self.k

    def flops(self) -> float:
        """GEMM flops of one step: gate/up 4RHI plus down 2RHI."""
        return 6.0 * self.R * self.H * self.I


WORKLOADS = {
    "tiny": Workload("tiny", 64, 256, 128, 8, 2, 0),
    "mixtral": Workload("mixtral", 4096, 4096, 14336, 8, 2, 1),
    "qwen3": Workload("qwen3", 8192, 2048, 768, 128, 8, 2, zipf=1.1),
    "dsv3_prefill": Workload("dsv3_prefill", 16384, 7168, 2048, 32, 8, 3, zipf=1.2),
    "dsv3_decode": Workload("dsv3_decode", 256, 7168, 2048, 32, 8, 4, wdtype="fp8"),
    # dsv3_prefill's and dsv3_decode's batches with fp8 weights and fp8 activations
    "dsv3_prefill_w8a8": Workload("dsv3_prefill_w8a8", 16384, 7168, 2048, 32, 8, 3, zipf=1.2,
                                  wdtype="fp8", act8=True),
    "dsv3_decode_w8a8": Workload("dsv3_decode_w8a8", 256, 7168, 2048, 32, 8, 4, wdtype="fp8",
                                 act8=True),
}


def bf16_bits_from_f32(a: np.ndarray) -> np.ndarray:
    """Round fp32 to bf16 (nearest, ties to even) and return the uint16 bits.

    Inputs are finite by construction (no NaN handling needed here)."""
    u = np.ascontiguousarray(a, dtype=np.float32).view(np.uint32)
    r = (u + np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1))) >> np.uint32(16)
    return r.astype(np.uint16)


def fp8e4m3_quantize_blocks(w: np.ndarray, block: int = 128):
    """Quantise an fp32 [N,K] matrix to fp8-e4m3fn with one fp32 scale per
    block x block tile: s = amax/448 (1 for an all-zero tile), q = RNE(w/s).

    Returns (q bits uint8 [N,K], scales fp32 [N/block, K/block])."""
    import torch  # CPU only; its fp8 cast is round-to-nearest-even

    n, kk = w.shape
    assert n % block == 0 and kk % block == 0
    t = w.reshape(n // block, block, kk // block, block)
    amax = np.abs(t).max(axis=(1, 3)).astype(np.float32)
    s = np.where(amax > 0, amax / np.float32(448.0), np.float32(1.0)).astype(np.float32)
    scaled = (t / s[:, None, :, None]).astype(np.float32).reshape(n, kk)
    q = torch.from_numpy(scaled).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    return np.ascontiguousarray(q), s


def route_tokens(logits: np.ndarray, k: int):
    """Client-side router: softmax, top-k (descending logit, ties to the lower
    id), renormalised weights. Returns (ids int32 [T,k], weights fp32 [T,k])."""
    order = np.argsort(-logits, axis=1, kind="stable")[:, :k]
    m = logits.max(axis=1, keepdims=True)
    p = np.exp(logits - m)
    p /= p.sum(axis=1, keepdims=True)
    psel = np.take_along_axis(p, order, axis=1)
    w = (psel / psel.sum(axis=1, keepdims=True)).astype(np.float32)
    return order.astype(np.int32), w


def _threads() -> int:
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def _expert_matrix(ss: np.random.SeedSequence, rows: int, cols: int, wdtype: str):
    g = np.random.Generator(np.random.PCG64(ss))
    a = g.standard_normal((rows, cols), dtype=np.float32)
    a *= np.float32(1.0 / np.sqrt(cols))
    if wdtype == "bf16":
        return bf16_bits_from_f32(a), None
    return fp8e4m3_quantize_blocks(a)


def _weights(ss: np.random.SeedSequence, E: int, rows: int, cols: int, wdtype: str):
    children = ss.spawn(E)
    with ThreadPoolExecutor(_threads()) as ex:
        parts = list(ex.map(lambda c: _expert_matrix(c, rows, cols, wdtype), children))
    w = np.stack([p[0] for p in parts])
    s = None if wdtype == "bf16" else np.stack([p[1] for p in parts])
    return w, s


def make_inputs(T: int, H: int, I: int, E: int, k: int, seed: int,
                zipf: float | None = None, wdtype: str = "bf16",
                weights: bool = True) -> dict:
    """Build one request batch plus the server's resident weights."""
    if wdtype not in ("bf16", "fp8"):
        raise ValueError(wdtype)
    s_x, s_gu, s_dn, s_lg, s_rk = np.random.SeedSequence(seed).spawn(5)
    gx = np.random.Generator(np.random.PCG64(s_x))
    x = bf16_bits_from_f32(gx.standard_normal((T, H), dtype=np.float32))
    logits = np.random.Generator(np.random.PCG64(s_lg)).standard_normal((T, E))
    if zipf is not None:
        rank = np.random.Generator(np.random.PCG64(s_rk)).permutation(E) + 1
        logits = logits + (-float(zipf) * np.log(rank.astype(np.float64)))[None, :]
    ids, w = route_tokens(logits, k)
    out = dict(T=T, H=H, I=I, E=E, k=k, wdtype=wdtype, x=x, topk_ids=ids,
               topk_weights=w)
    if weights:
        wgu, sgu = _weights(s_gu, E, 2 * I, H, wdtype)
        wdn, sdn = _weights(s_dn, E, H, I, wdtype)
        out.update(w_gate_up=wgu, w_gate_up_scale=sgu, w_down=wdn, w_down_scale=sdn)
    return out


def make_workload(name: str, weights: bool = True) -> dict:
    wl = WORKLOADS[name]
    d = make_inputs(wl.T, wl.H, wl.I, wl.E, wl.k, wl.seed, wl.zipf, wl.wdtype, weights)
    d["workload"] = asdict(wl)
    d["act8"] = wl.act8
    return d


def manifest(inputs: dict) -> dict:
    """SHA-256 of every array (used to pin generator determinism)."""
    return {key: hashlib.sha256(np.ascontiguousarray(v).tobytes()).hexdigest()
            for key, v in sorted(inputs.items()) if isinstance(v, np.ndarray)}
