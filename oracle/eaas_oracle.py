"""Plain, slow CPU oracle for one stateless expert server's forward step.

TEST INFRASTRUCTURE ONLY.  Imported by ``tests/``, ``__graft_entry__.smoke()``
and the cpu_baseline leg of ``bench.py``; nothing in the product library
imports, links or runs it, and it shares no code with the HIP path.

What it computes (EaaS, §3.3 "Asynchronous Server Operation"): the server takes
the payload of a request (§3.2: hidden states, an expert id per token slot and
the router score used to weight outputs), regroups the token slots by expert,
runs every resident expert's FFN over its rows, and returns for each token the
router-score-weighted sum of its experts' outputs.  The regrouping is the
"token reorganization" of §3.3 and Fig. 5; the list of non-empty experts is the
compacted active-group list produced by the group-shrink prefix scan of §4.1.

Readings (the paper does not define the FFN or precisions):
  * FFN = SwiGLU without bias: y = W_down (silu(W_gate x) * (W_up x)), with
    W_gate_up[e] = [W_gate; W_up] stacked on rows ([0,I) gate, [I,2I) up) and
    every weight stored [out, in] row-major.
  * Slot s = t*k + j is valid iff 0 <= ids[s] < E; invalid slots are skipped
    (ids of experts living on other servers).
  * Rows inside an expert's segment are in ascending slot order (the unique
    stable counting sort), so perm/inv/offsets are defined bit-exactly.
  * G and U are accumulated in fp64 from the exact bf16 (or dequantised fp8)
    operands; the intermediate h is stored in bf16: h = bf16_rne(silu(g)*u)
    evaluated in fp32 from g = fp32(G), u = fp32(U) -- the precision at which
    the kernel takes that rounding decision.  The down projection and the
    weighted sum (ascending j, from +0) are fp64.
  * fp8 weights are OCP e4m3fn with one fp32 scale per 128x128 block of each
    expert matrix; dequantisation is W = fp32(q) * s, one fp32 rounding.
"""
from __future__ import annotations

import numpy as np

__all__ = [
    "bf16_to_f32", "f32_to_bf16_rne", "e4m3fn_to_f32", "dequantize_blocks",
    "route_permute", "silu_mul_to_bf16", "expert_ffn_grouped",
    "unpermute_combine", "expert_forward", "brute_force_tokens",
    "weights_f32", "expert_weights_f64", "sub_batch",
]


# --------------------------------------------------------------------------
# number formats
# --------------------------------------------------------------------------
def bf16_to_f32(bits: np.ndarray) -> np.ndarray:
    """bf16 bit pattern -> fp32 (exact: bf16 is the top half of fp32)."""
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def f32_to_bf16_rne(a: np.ndarray) -> np.ndarray:
    """fp32 -> bf16 bits, round to nearest, ties to even; NaN stays NaN."""
    a = np.asarray(a, dtype=np.float32)
    u = a.view(np.uint32).astype(np.uint64)
    lsb = (u >> np.uint64(16)) & np.uint64(1)
    r = ((u + np.uint64(0x7FFF) + lsb) >> np.uint64(16)).astype(np.uint16)
    nan = np.isnan(a)
    if nan.any():
        r = np.where(nan, ((u >> np.uint64(16)) | np.uint64(0x40)).astype(np.uint16), r)
    return r


def e4m3fn_to_f32(bits: np.ndarray) -> np.ndarray:
    """OCP fp8 e4m3fn bits -> fp32.  1 sign, 4 exponent (bias 7), 3 mantissa
    bits; exponent 0 is subnormal (m * 2^-9); S.1111.111 is NaN; no infinity."""
    b = np.asarray(bits, dtype=np.uint8).astype(np.int32)
    sign = np.where(b & 0x80, -1.0, 1.0)
    e = (b >> 3) & 0xF
    m = b & 0x7
    normal = np.ldexp(1.0 + m / 8.0, e - 7)
    sub = np.ldexp(m.astype(np.float64), -9)
    v = sign * np.where(e == 0, sub, normal)
    v = np.where((e == 15) & (m == 7), np.nan, v)
    return v.astype(np.float32)


def dequantize_blocks(q: np.ndarray, s: np.ndarray, block: int = 128) -> np.ndarray:
    """W[r, c] = fp32(q[r, c]) * s[r // block, c // block], one fp32 rounding."""
    w = e4m3fn_to_f32(q)
    srep = np.repeat(np.repeat(np.asarray(s, np.float32), block, axis=-2), block, axis=-1)
    return (w * srep).astype(np.float32)


def weights_f32(inp: dict):
    """Dequantised fp32 weights of all experts (exact for bf16) as
    (W_gate_up [E,2I,H], W_down [E,H,I])."""
    if inp["wdtype"] == "bf16":
        return bf16_to_f32(inp["w_gate_up"]), bf16_to_f32(inp["w_down"])
    return (dequantize_blocks(inp["w_gate_up"], inp["w_gate_up_scale"]),
            dequantize_blocks(inp["w_down"], inp["w_down_scale"]))


def expert_weights_f64(inp: dict, e: int, weights=None):
    """(W_gate [I,H], W_up [I,H], W_down [H,I]) of expert e as fp64, converted
    one expert at a time so full-size weights never exist in fp64 at once."""
    I = inp["I"]
    if weights is not None:
        wgu, wdn = weights[0][e], weights[1][e]
    elif inp["wdtype"] == "bf16":
        wgu, wdn = bf16_to_f32(inp["w_gate_up"][e]), bf16_to_f32(inp["w_down"][e])
    else:
        wgu = dequantize_blocks(inp["w_gate_up"][e], inp["w_gate_up_scale"][e])
        wdn = dequantize_blocks(inp["w_down"][e], inp["w_down_scale"][e])
    wgu = np.asarray(wgu, dtype=np.float64)
    return wgu[:I], wgu[I:], np.asarray(wdn, dtype=np.float64)


def sub_batch(inp: dict, tokens) -> dict:
    """The request restricted to some tokens.  Expert outputs of a token depend
    on that token alone (the server is stateless, §2.4), so the step applied to
    the sub-batch gives exactly those tokens' rows of the full result."""
    tokens = np.asarray(list(tokens), dtype=np.int64)
    d = dict(inp)
    d.update(T=int(tokens.size), x=inp["x"][tokens], topk_ids=inp["topk_ids"][tokens],
             topk_weights=inp["topk_weights"][tokens])
    return d


# --------------------------------------------------------------------------
# token reorganisation (§3.3) and group-shrink compaction (§4.1)
# --------------------------------------------------------------------------
def route_permute(topk_ids: np.ndarray, E: int) -> dict:
    """Group the T*k token slots by expert with a stable counting sort.

    counts[e]   number of valid slots with id e
    offsets     exclusive prefix sum of counts, length E+1
    perm[r]     flat slot s = t*k+j held by row r (rows >= offsets[E]: -1)
    inv[s]      row of slot s, or -1 for an invalid slot
    active      [n_active, e_1 < e_2 < ...] experts with a non-zero count
    """
    ids = np.asarray(topk_ids, dtype=np.int64).reshape(-1)
    R = ids.size
    valid = (ids >= 0) & (ids < E)
    counts = np.bincount(ids[valid], minlength=E).astype(np.int32)
    offsets = np.zeros(E + 1, dtype=np.int32)
    offsets[1:] = np.cumsum(counts)
    slots = np.flatnonzero(valid)
    order = np.argsort(ids[slots], kind="stable")
    perm = np.full(R, -1, dtype=np.int32)
    perm[: slots.size] = slots[order]
    inv = np.full(R, -1, dtype=np.int32)
    inv[perm[: slots.size]] = np.arange(slots.size, dtype=np.int32)
    act = np.flatnonzero(counts > 0).astype(np.int32)
    active = np.zeros(E + 1, dtype=np.int32)
    active[0] = act.size
    active[1: 1 + act.size] = act
    return dict(counts=counts, offsets=offsets, perm=perm, inv=inv, active=active)


# --------------------------------------------------------------------------
# expert FFN over the grouped rows
# --------------------------------------------------------------------------
def silu_mul_to_bf16(G: np.ndarray, U: np.ndarray) -> np.ndarray:
    """h = bf16_rne(silu(g) * u) with g, u, silu and the product in fp32."""
    g = np.asarray(G, dtype=np.float32)
    u = np.asarray(U, dtype=np.float32)
    with np.errstate(over="ignore"):
        s = g / (np.float32(1.0) + np.exp(-g))
    return f32_to_bf16_rne((s * u).astype(np.float32))


def expert_ffn_grouped(inp: dict, routing: dict, weights=None):
    """Per active expert e: rows r in [offsets[e], offsets[e+1]) hold token
    t_r = perm[r] // k; y[r] = W_down[e] h_r with h_r as in silu_mul_to_bf16.
    Returns (h bits uint16 [R, I], y fp64 [R, H]); rows past offsets[E] are 0."""
    T, H, I, k = inp["T"], inp["H"], inp["I"], inp["k"]
    R = T * k
    x = bf16_to_f32(inp["x"]).astype(np.float64)
    off, perm, active = routing["offsets"], routing["perm"], routing["active"]
    h = np.zeros((R, I), dtype=np.uint16)
    y = np.zeros((R, H), dtype=np.float64)
    for e in active[1: 1 + active[0]]:
        r0, r1 = int(off[e]), int(off[e + 1])
        A = x[perm[r0:r1] // k]
        Wg, Wu, Wd = expert_weights_f64(inp, int(e), weights)
        G = A @ Wg.T
        U = A @ Wu.T
        hb = silu_mul_to_bf16(G, U)
        h[r0:r1] = hb
        y[r0:r1] = bf16_to_f32(hb).astype(np.float64) @ Wd.T
    return h, y


def unpermute_combine(y: np.ndarray, routing: dict, topk_weights: np.ndarray) -> np.ndarray:
    """out[t] = sum over ascending j of w[t, j] * y[inv[t*k+j]] for valid
    slots, starting from +0; a token without a valid slot gets zeros."""
    T, k = topk_weights.shape
    inv = routing["inv"].reshape(T, k)
    w = topk_weights.astype(np.float64)
    out = np.zeros((T, y.shape[1]), dtype=np.float64)
    for j in range(k):
        v = inv[:, j] >= 0
        rows = np.where(v, inv[:, j], 0)
        out += np.where(v[:, None], w[:, j, None] * y[rows], 0.0)
    return out


def expert_forward(inp: dict, weights=None) -> dict:
    """The whole step: routing, grouped SwiGLU FFN, weighted combine."""
    routing = route_permute(inp["topk_ids"], inp["E"])
    h, y = expert_ffn_grouped(inp, routing, weights)
    out = unpermute_combine(y, routing, inp["topk_weights"])
    return dict(routing=routing, h=h, y=y, out=out)


# --------------------------------------------------------------------------
# token-by-token brute force: dense evaluation of every selected expert
# --------------------------------------------------------------------------
def brute_force_tokens(inp: dict, tokens, weights=None, mirror_h: bool = True) -> np.ndarray:
    """For each requested token t: sum_j w[t,j] * FFN_{ids[t,j]}(x_t) in fp64,
    evaluated directly from the definition with no grouping.  With
    mirror_h=True the intermediate is rounded as in silu_mul_to_bf16; with
    mirror_h=False it is the exact fp64 SwiGLU."""
    E, H = inp["E"], inp["H"]
    ids, w = inp["topk_ids"], inp["topk_weights"]
    tokens = list(tokens)
    cache = {}
    out = np.zeros((len(tokens), H), dtype=np.float64)
    for n, t in enumerate(tokens):
        xt = bf16_to_f32(inp["x"][t]).astype(np.float64)
        for j in range(ids.shape[1]):
            e = int(ids[t, j])
            if not (0 <= e < E):
                continue
            if e not in cache:
                cache[e] = expert_weights_f64(inp, e, weights)
            Wg, Wu, Wd = cache[e]
            g = Wg @ xt
            u = Wu @ xt
            if mirror_h:
                hv = bf16_to_f32(silu_mul_to_bf16(g, u)).astype(np.float64)
            else:
                hv = g / (1.0 + np.exp(-g)) * u
            out[n] += float(w[t, j]) * (Wd @ hv)
    return out
