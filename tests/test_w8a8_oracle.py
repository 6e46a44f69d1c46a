"""Pins of the fp8-weight / fp8-activation oracle (no GPU).

The e4m3fn quantizer is pinned to torch's float8_e4m3fn cast (a library
routine) and to the format itself (every code round-trips; ties go to the
even code; saturation at 448).  The per-(row, 128-channel) scales are pinned
by closed forms: an all-zero block has scale 1, the largest magnitude of a
block maps to the code of 448, and the dequantized error stays within half a
spacing.  The step is pinned by a special case that reduces to the
fp8-weight step: when every activation block is already on the e4m3 grid
with a power-of-two scale, the quantization is exact, so G, U and h equal
that step's bit for bit.  The error against the unquantized step is bounded
by the fp8 grid.  The planted-mistake tests show a slip in the scales or the
blocking fails a pin.
"""
import numpy as np
import pytest
import torch

from oracle import eaas_oracle as O
from oracle import w8a8_oracle as W
from paper_2509_17863_amd import synth


def finite_codes():
    return np.array([c for c in range(256) if (c & 0x7F) != 0x7F], dtype=np.uint8)


# ----------------------------------------------------------------- quantizer
def test_every_code_round_trips():
    c = finite_codes()
    assert np.array_equal(W.f32_to_e4m3fn_rne(O.e4m3fn_to_f32(c)), c)


def test_quantizer_matches_torch_cast():
    rng = np.random.default_rng(3)
    v = O.e4m3fn_to_f32(finite_codes()).astype(np.float64)
    pos = np.unique(v[v > 0])
    mids = (pos[:-1] + pos[1:]) / 2           # exact ties between neighbours
    x = np.concatenate([rng.standard_normal(100000) * s for s in (1e-3, 0.05, 1.0, 30.0, 300.0)]
                       + [mids, -mids, pos, -pos, [0.0, -0.0]]).astype(np.float32)
    x = x[np.abs(x) <= 448]
    ref = torch.from_numpy(x).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    assert np.array_equal(W.f32_to_e4m3fn_rne(x), ref)


def test_ties_go_to_even_and_saturate():
    # 1.0625 lies between 1.0 (code 0x38, even mantissa) and 1.125 (0x39)
    assert W.f32_to_e4m3fn_rne(np.float32(1.0625)) == 0x38
    # 1.1875 lies between 1.125 (0x39) and 1.25 (0x3A, even)
    assert W.f32_to_e4m3fn_rne(np.float32(1.1875)) == 0x3A
    # subnormal tie: 1.5 * 2^-9 between 2^-9 (0x01) and 2^-8 (0x02, even)
    assert W.f32_to_e4m3fn_rne(np.float32(1.5 * 2.0 ** -9)) == 0x02
    # below half the smallest subnormal: zero, with its sign
    assert W.f32_to_e4m3fn_rne(np.float32(-0.4 * 2.0 ** -9)) == 0x80
    # past the largest finite value: saturate, never NaN
    big = np.array([448.0, 463.0, 464.0, 1e6, -1e30], dtype=np.float32)
    assert W.f32_to_e4m3fn_rne(big).tolist() == [0x7E, 0x7E, 0x7E, 0x7E, 0xFE]


# ----------------------------------------------------------------- row-block scales
def test_row_block_scales_closed_forms():
    rng = np.random.default_rng(5)
    a = rng.standard_normal((6, 384)).astype(np.float32) * np.float32(3.0)
    a[2, 128:256] = 0.0                       # an all-zero block
    q, s = W.quantize_rows_blocks(a)
    assert s.shape == (6, 3) and q.shape == a.shape
    assert s[2, 1] == 1.0 and np.all(q[2, 128:256] == 0)
    amax = np.abs(a.reshape(6, 3, 128)).max(axis=2)
    nz = amax > 0
    assert np.array_equal(s[nz], (amax[nz] / np.float32(448.0)).astype(np.float32))
    # the largest magnitude of each block lands on +-448
    blk = a.reshape(6, 3, 128)
    qb = q.reshape(6, 3, 128)
    for r in range(6):
        for b in range(3):
            if nz[r, b]:
                i = int(np.abs(blk[r, b]).argmax())
                assert qb[r, b, i] & 0x7F == 0x7E
    # dequantized error within half a spacing of the e4m3 grid (relative 2^-4
    # for normals, 2^-10 * s absolute for subnormals)
    d = W.dequantize_rows_blocks(q, s).reshape(6, 3, 128)
    srep = s[:, :, None].astype(np.float64)
    bound = np.maximum(np.abs(blk) * 2.0 ** -4, srep * 2.0 ** -10) * (1 + 1e-6)
    assert np.all(np.abs(d - blk) <= bound)


# ----------------------------------------------------------------- the step
def grid_inputs(T=24, H=256, I=128, E=3, k=2, seed=21):
    """fp8 weights with power-of-two block scales and activations whose every
    128-block is an e4m3 value times a power of two, with max |.| = 448 * 2^m:
    both quantizations are exact."""
    d = synth.make_inputs(T, H, I, E, k, seed, wdtype="fp8")
    rng = np.random.default_rng(seed)
    codes = finite_codes()
    vals = O.e4m3fn_to_f32(codes).astype(np.float64)
    vals = vals[np.abs(vals) <= 448]
    x = rng.choice(vals, size=(T, H // 128, 128))
    x[:, :, 0] = 448.0                        # pin each block's amax to 448
    m = rng.integers(-9, -4, size=(T, H // 128, 1))
    x = (x * np.ldexp(1.0, m)).reshape(T, H)  # scale 2^m exactly, still bf16-exact
    d["x"] = synth.bf16_bits_from_f32(x.astype(np.float32))
    assert np.array_equal(O.bf16_to_f32(d["x"]).astype(np.float64), x)
    for key in ("w_gate_up_scale", "w_down_scale"):
        d[key] = np.ldexp(1.0, np.round(np.log2(d[key])).astype(np.int64)).astype(np.float32)
    return d


def test_exact_grid_reduces_to_fp8_weight_step():
    d = grid_inputs()
    r8 = W.expert_forward_w8a8(d)
    ref = O.expert_forward(d)
    # x is on the grid: its quantization is the identity
    assert np.array_equal(W.dequantize_rows_blocks(r8["xq"], r8["sx"]),
                          O.bf16_to_f32(d["x"]).astype(np.float64))
    # so G, U, and the bf16 intermediate are the fp8-weight step's
    assert np.array_equal(r8["h"], ref["h"])
    # and the down input is h quantized per row block
    hq, sh = W.quantize_rows_blocks(O.bf16_to_f32(ref["h"]))
    assert np.array_equal(r8["hq"], hq) and np.array_equal(r8["sh"], sh)


def test_error_against_unquantized_step_is_fp8_sized():
    d = synth.make_inputs(48, 512, 256, 4, 2, seed=31, wdtype="fp8")
    r8 = W.expert_forward_w8a8(d)
    ref = O.expert_forward(d)
    rms = np.sqrt((ref["out"] ** 2).mean())
    rel = np.sqrt(((r8["out"] - ref["out"]) ** 2).mean()) / rms
    # two fp8 roundings (relative spacing 2^-3, uniform error ~2.5% rms each)
    # averaged over K: a few percent, and not zero
    assert 0.003 < rel < 0.08, rel


# ----------------------------------------------------------------- planted mistakes
def _pins():
    yield test_exact_grid_reduces_to_fp8_weight_step
    yield test_error_against_unquantized_step_is_fp8_sized
    yield test_row_block_scales_closed_forms


def _mutants():
    real_q = W.quantize_rows_blocks
    real_dq = W.dequantize_rows_blocks
    real_w = W._weights_f64

    def scales_shifted(q, s, block=128):           # block b uses the scale of b+1
        return real_dq(q, np.roll(s, -1, axis=1), block)

    def scale_not_applied(q, s, block=128):
        return real_dq(q, np.ones_like(s), block)

    def amax_over_row(a, block=128):               # one scale per row, not per block
        q, s = real_q(a, a.shape[1])
        return q, np.repeat(s, a.shape[1] // block, axis=1)

    def weight_scale_transposed(q, s, block=128):
        return real_w(q, np.ascontiguousarray(s.T) if s.shape[0] == s.shape[1] else s[::-1], block)

    return [("dequantize_rows_blocks", scales_shifted), ("dequantize_rows_blocks", scale_not_applied),
            ("quantize_rows_blocks", amax_over_row), ("_weights_f64", weight_scale_transposed)]


@pytest.mark.parametrize("idx", range(4))
def test_planted_mistake_is_caught(monkeypatch, idx):
    name, fn = _mutants()[idx]
    monkeypatch.setattr(W, name, fn)
    caught = 0
    for pin in _pins():
        try:
            pin()
        except AssertionError:
            caught += 1
    assert caught >= 1, f"no pin caught the planted mistake in {name}"
