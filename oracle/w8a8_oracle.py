"""CPU oracle for the expert step with fp8 weights AND fp8 activations.

TEST INFRASTRUCTURE ONLY.  Imported by ``tests/`` (and through ``oracle``);
nothing in the product library imports, links or runs it, and it shares no
code with the HIP path.

The paper names DeepGEMM as the grouped-GEMM engine (§4.1) without fixing
precisions.  This mode follows the block-scaled fp8 recipe that engine is
built for.  The weights keep the fp8 format of the fp8-weight step: OCP
e4m3fn with one fp32 scale per 128x128 block.  The activations entering
each grouped GEMM are quantized too, per row and per 128 consecutive
channels:

    s = amax(|a|) / 448 over the 128 values (s = 1 when they are all 0),
    q = e4m3fn_rne_sat(a / s)

s and a/s are evaluated in fp32 (that is where the code is decided), and the
conversion rounds to nearest, ties to even, saturating at +-448.  The step
is:
  * gate/up input: x (bf16, exact in fp32), quantized per token;
  * G, U = dequant(xq) . dequant(W_gate_up)^T, exactly (in fp64);
  * h = bf16_rne(silu(fp32 G) * fp32 U), as in the bf16 step;
  * down input: h (as fp32), quantized per row of the grouped layout;
  * y = dequant(hq) . dequant(W_down)^T in fp64, then the weighted combine.
Dequantization here is exact: fp64(q) * fp64(s).

Readings where the paper is silent (binding for the library as well):
  * quantization blocks are 128 channels along K, one per (row, block), the
    same K blocking as the weights, so that a 128-wide K block has a single
    activation scale and a single weight scale;
  * NaN inputs give NaN codes (0x7f with the sign); the inputs of this
    build are finite.
"""
from __future__ import annotations

import numpy as np

from .eaas_oracle import (bf16_to_f32, e4m3fn_to_f32, route_permute, silu_mul_to_bf16,
                          unpermute_combine)

__all__ = ["E4M3_MAX", "f32_to_e4m3fn_rne", "quantize_rows_blocks", "dequantize_rows_blocks",
           "expert_forward_w8a8"]

E4M3_MAX = 448.0


def f32_to_e4m3fn_rne(a: np.ndarray) -> np.ndarray:
    """fp32 -> OCP fp8 e4m3fn bits, round to nearest even, saturating.

    The format (1 sign, 4 exponent bits with bias 7, 3 mantissa bits) has
    normal values (1 + m/8) * 2^(e-7) for e in 1..15 (except S.1111.111,
    which is NaN) and subnormals m * 2^-9.  So on [2^n, 2^(n+1)) with
    n >= -6 the spacing is 2^(n-3), and below 2^-6 it is 2^-9.  A magnitude
    is divided by its spacing, rounded half to even, and multiplied back
    (all exact in fp64); results past 448 saturate to 448."""
    x = np.asarray(a, dtype=np.float32).astype(np.float64)
    mag = np.abs(x)
    _, ex = np.frexp(mag)                       # mag = f * 2^ex, f in [0.5, 1)
    n = np.maximum(ex - 1, -6)                  # binade (floor log2), clamped to the normals
    step = np.ldexp(1.0, n - 3)
    r = np.minimum(np.rint(mag / step) * step, E4M3_MAX)
    _, er = np.frexp(r)
    nr = er - 1                                 # binade of the rounded value (may carry up)
    normal = (r > 0) & (nr >= -6)
    code_norm = ((nr + 7) << 3) | np.rint((np.ldexp(r, -nr) - 1.0) * 8.0).astype(np.int64)
    code_sub = np.rint(np.ldexp(r, 9)).astype(np.int64)
    code = np.where(normal, code_norm, code_sub)
    sign = np.signbit(x).astype(np.int64) << 7
    out = (code | sign).astype(np.uint8)
    return np.where(np.isnan(x), (sign | 0x7F).astype(np.uint8), out)


def quantize_rows_blocks(a: np.ndarray, block: int = 128):
    """a [rows, K] (fp32 values) -> (q uint8 [rows, K], s fp32 [rows, K/block]):
    per row and per block of `block` channels, s = amax/448 in fp32 (1 for
    an all-zero block) and q = e4m3fn_rne(a / s) with the quotient in fp32."""
    a = np.asarray(a, dtype=np.float32)
    rows, K = a.shape
    assert K % block == 0
    b = a.reshape(rows, K // block, block)
    amax = np.abs(b).max(axis=2)
    s = np.where(amax > 0, amax / np.float32(E4M3_MAX), np.float32(1.0)).astype(np.float32)
    scaled = (b / s[:, :, None]).astype(np.float32)
    return f32_to_e4m3fn_rne(scaled).reshape(rows, K), s


def dequantize_rows_blocks(q: np.ndarray, s: np.ndarray, block: int = 128) -> np.ndarray:
    """Exact fp64 values of row-block-quantized data: fp64(q) * fp64(s)."""
    v = e4m3fn_to_f32(q).astype(np.float64)
    rows, K = v.shape
    return (v.reshape(rows, K // block, block) * np.asarray(s, np.float64)[:, :, None]).reshape(rows, K)


def _weights_f64(q: np.ndarray, s: np.ndarray, block: int = 128) -> np.ndarray:
    """Exact fp64 values of one expert's block-quantized [N, K] weights."""
    v = e4m3fn_to_f32(q).astype(np.float64)
    srep = np.repeat(np.repeat(np.asarray(s, np.float64), block, axis=0), block, axis=1)
    return v * srep


def expert_forward_w8a8(inp: dict) -> dict:
    """The step with fp8 weights and fp8 activations (module docstring).
    Returns routing, xq/sx (the quantized x), hq/sh (the quantized h in the
    grouped row order), h (bf16 bits before its quantization), y and out."""
    assert inp["wdtype"] == "fp8"
    T, H, I, E, k = inp["T"], inp["H"], inp["I"], inp["E"], inp["k"]
    R = T * k
    routing = route_permute(inp["topk_ids"], E)
    xq, sx = quantize_rows_blocks(bf16_to_f32(inp["x"]))
    xd = dequantize_rows_blocks(xq, sx)
    off, perm, active = routing["offsets"], routing["perm"], routing["active"]
    h = np.zeros((R, I), dtype=np.uint16)
    hq = np.zeros((R, I), dtype=np.uint8)
    sh = np.ones((R, I // 128), dtype=np.float32)
    y = np.zeros((R, H), dtype=np.float64)
    for e in active[1: 1 + active[0]]:
        e = int(e)
        r0, r1 = int(off[e]), int(off[e + 1])
        A = xd[perm[r0:r1] // k]
        wgu = _weights_f64(inp["w_gate_up"][e], inp["w_gate_up_scale"][e])
        G = A @ wgu[:I].T
        U = A @ wgu[I:].T
        hb = silu_mul_to_bf16(G, U)
        h[r0:r1] = hb
        q, s = quantize_rows_blocks(bf16_to_f32(hb))
        hq[r0:r1], sh[r0:r1] = q, s
        wd = _weights_f64(inp["w_down"][e], inp["w_down_scale"][e])
        y[r0:r1] = dequantize_rows_blocks(q, s) @ wd.T
    out = unpermute_combine(y, routing, inp["topk_weights"])
    return dict(routing=routing, xq=xq, sx=sx, h=h, hq=hq, sh=sh, y=y, out=out)
