"""GPU parity of the fp8-weight, fp8-activation step (EAAS_FP8_E4M3_A8)
through the C ABI, against its CPU oracle, stage by stage.

1. The quantized x (codes and scales, read from the workspace) must equal the
   oracle's bit for bit: the same inputs, the same fp32 arithmetic.
2. h is quantized from the kernel's own h, whose fp32 accumulation (and
   hardware exp) differs from the oracle's fp64 h by at most a bound derived
   from the fp32 sums (h_bounds).  So each 128-block of the kernel's h codes
   must be a valid quantization of an h' within that distance of the
   oracle's h: its scale between the smallest and largest amax/448 such an
   h' allows, every code between the codes of h_ref -+ that distance.  Codes
   may differ from the oracle's own in a few places; when a block's
   maximum lands one ulp apart, its scale moves and many of its codes with
   it, so a plain comparison of codes would reject correct results.
3. The output must equal the oracle's down projection and weighted sum of the
   kernel's own quantized h within max|gpu - ref| <= 2e-2 * RMS(ref).
4. End to end against the oracle, the RMS of the error stays below
   2e-2 * RMS (single code flips near a block maximum move single outputs
   by a few percent of the RMS, so the maximum is not bounded this way).
Every case prints its name before touching the GPU.
"""
import numpy as np
import pytest
import torch

from oracle import eaas_oracle as O
from oracle import w8a8_oracle as W
from paper_2509_17863_amd import eaas, synth
from paper_2509_17863_amd.device_io import to_device

pytestmark = pytest.mark.gpu

TOL = 2e-2


def say(*a):
    print("[gpu-case]", *a, flush=True)


def gpu_quantize(x_bits):
    rows, K = x_bits.shape
    x = torch.from_numpy(x_bits.view(np.int16)).cuda()
    q = torch.empty((rows, K), dtype=torch.uint8, device="cuda")
    s = torch.empty((rows, K // 128), dtype=torch.float32, device="cuda")
    eaas.eaas_quantize_rows_fp8(x, q, s)
    torch.cuda.synchronize()
    return q.cpu().numpy(), s.cpu().numpy()


def check_quant_bitexact(x_bits, what):
    say("quantize", what, x_bits.shape)
    q, s = gpu_quantize(x_bits)
    rq, rs = W.quantize_rows_blocks(O.bf16_to_f32(x_bits))
    assert np.array_equal(s.view(np.uint32), rs.view(np.uint32)), f"{what}: scales"
    bad = np.flatnonzero(q.ravel() != rq.ravel())
    assert bad.size == 0, f"{what}: {bad.size} codes differ, first at {bad[:5]}"


@pytest.mark.parametrize("rows,K,scale,seed", [(37, 384, 1.0, 0), (5, 128, 1e-3, 1),
                                               (300, 1024, 40.0, 2), (1, 7168, 1.0, 3)])
def test_quantize_rows_bitexact(gpu, rows, K, scale, seed):
    rng = np.random.default_rng(seed)
    x = (rng.standard_normal((rows, K)) * scale).astype(np.float32)
    x[:, :128] *= np.float32(1e-3)          # small values: subnormal e4m3 codes
    if rows > 2:
        x[2, 128:256] = 0.0                 # an all-zero block (scale 1)
    check_quant_bitexact(synth.bf16_bits_from_f32(x), f"random {rows}x{K}")


def test_quantize_rows_ties_and_edges(gpu):
    # blocks with amax 448 have scale exactly 1: the values are then quantized
    # as they are, so midpoints between e4m3 neighbours are exact ties
    codes = np.array([c for c in range(256) if (c & 0x7F) != 0x7F], dtype=np.uint8)
    vals = O.e4m3fn_to_f32(codes).astype(np.float64)
    pos = np.unique(vals[vals > 0])
    mids = (pos[:-1] + pos[1:]) / 2
    mids = mids[O.bf16_to_f32(synth.bf16_bits_from_f32(mids.astype(np.float32))) == mids]
    body = np.concatenate([mids, -mids, pos, -pos, [0.0, -0.0]])
    n = int(np.ceil(body.size / 127))
    x = np.zeros((n, 128), dtype=np.float64)
    x[:, 0] = 448.0
    flat = np.zeros(n * 127)
    flat[: body.size] = body
    x[:, 1:] = flat.reshape(n, 127)
    check_quant_bitexact(synth.bf16_bits_from_f32(x.astype(np.float32)), "ties and edges")


def forward_a8(d, out_dtype=torch.float32):
    dev = to_device(d)
    T, H = dev["x"].shape
    E, twoI, _ = dev["w_gate_up"].shape
    k = d["k"]
    ws = eaas.alloc_workspace(T, H, twoI // 2, E, k, eaas.EAAS_FP8_E4M3_A8)
    out = torch.full((T, H), float("nan"), dtype=out_dtype, device="cuda")
    eaas.eaas_expert_forward(dev["x"], dev["topk_ids"], dev["topk_weights"], dev["w_gate_up"],
                             dev["w_down"], out, ws, dev["w_gate_up_scale"],
                             dev["w_down_scale"], act8=True)
    torch.cuda.synchronize()
    return out.float().cpu().numpy(), ws


def ws_arrays(d, ws):
    """The quantized x and h the step left in its workspace."""
    T, H, I, E, k = d["T"], d["H"], d["I"], d["E"], d["k"]
    A8 = eaas.EAAS_FP8_E4M3_A8

    def view(region, dtype, shape):
        return eaas.workspace_view(ws, T, H, I, E, k, A8, region).cpu().numpy().view(dtype).reshape(shape)

    R = T * k
    return dict(xq=view(eaas.EAAS_WS_XQ, np.uint8, (T, H)),
                xs=view(eaas.EAAS_WS_XS, np.float32, (T, H // 128)),
                hq=view(eaas.EAAS_WS_HQ, np.uint8, (R, I)),
                hs=view(eaas.EAAS_WS_HS, np.float32, (R, I // 128)))


def check_close(got, ref, what):
    got = np.asarray(got, dtype=np.float64)
    rms = float(np.sqrt((ref ** 2).mean())) if ref.size else 0.0
    err = float(np.abs(got - ref).max()) if ref.size else 0.0
    say(f"{what}: max_abs_err={err:.3e} rms={rms:.3e} ratio={err / max(rms, 1e-30):.2e}")
    assert np.isfinite(got).all(), f"{what}: non-finite output"
    assert err <= TOL * rms, f"{what}: {err} > {TOL} * {rms}"


def bf16_ulp(v):
    m = np.maximum(np.abs(v).astype(np.float64), 2.0 ** -126)
    return np.ldexp(1.0, np.floor(np.log2(m)).astype(np.int64) - 7)


# The fp8 MFMAs do not sum their 64 products in full fp32: measured on this
# GPU (test_fp8_mfma_accumulation_error), a K tile's dot product errs by up
# to about 2^-14.7 of the sum of the magnitudes of its terms.  The bounds
# below allow 2^-12 (with the fp32 promotion across K tiles far below that).
MFMA_EPS = 2.0 ** -12


def h_bounds_rows(g, u, sg, su):
    """The oracle's bf16 h bits for rows with exact G, U (fp64) and a bound on
    how far the kernel's bf16 h may lie from it.  |dG| <= MFMA_EPS * sum|a w|
    (sg; likewise U, su); h = silu(g) u then moves by |silu'(g) u| |dG| +
    |silu(g)| |dU|, plus a few fp32 ulp for the hardware exp and reciprocal,
    plus one bf16 ulp for the two roundings."""
    eps = MFMA_EPS
    sig = 1.0 / (1.0 + np.exp(-g))
    dsilu = sig * (1.0 + g * (1.0 - sig))
    hb = O.silu_mul_to_bf16(g, u)
    hv = O.bf16_to_f32(hb).astype(np.float64)
    dh = np.abs(dsilu * u) * eps * sg + np.abs(g * sig) * eps * su + 2.0 ** -20 * np.abs(hv)
    return hb, dh + bf16_ulp(hv)


def check_h_quantization(h_bits, tol, hq, hs, what):
    """hq, hs [rows, I] of the kernel against the oracle's bf16 h [rows, I]
    (same rows): every block a valid quantization of an h' with
    |h' - h| <= tol elementwise (see module doc).  Returns how many codes
    differ from the oracle's own quantization of its h."""
    h = O.bf16_to_f32(h_bits).astype(np.float64)
    rows, I = h.shape
    hb = h.reshape(rows, I // 128, 128)
    tb = tol.reshape(rows, I // 128, 128)
    amax_lo = np.maximum(np.abs(hb) - tb, 0).max(axis=2)
    amax_hi = (np.abs(hb) + tb).max(axis=2)
    sg = hs.astype(np.float64)
    ok_s = (sg >= amax_lo / 448 * (1 - 2e-7)) & (sg <= amax_hi / 448 * (1 + 2e-7))
    ok_s |= (amax_lo == 0) & (sg == 1.0)
    assert ok_s.all(), f"{what}: {np.count_nonzero(~ok_s)} h scales out of bounds"
    s3 = hs.astype(np.float32)[:, :, None]
    lo = O.e4m3fn_to_f32(W.f32_to_e4m3fn_rne(((hb - tb).astype(np.float32) / s3).astype(np.float32)))
    hi = O.e4m3fn_to_f32(W.f32_to_e4m3fn_rne(((hb + tb).astype(np.float32) / s3).astype(np.float32)))
    got = O.e4m3fn_to_f32(hq.reshape(rows, I // 128, 128))
    ok = (got >= lo) & (got <= hi)
    assert ok.all(), f"{what}: {np.count_nonzero(~ok)} h codes are no quantization of a nearby h"
    ref_q, _ = W.quantize_rows_blocks(O.bf16_to_f32(h_bits))
    return int(np.count_nonzero(ref_q != hq))


def check_step(d, got, ws, what):
    """Every token of the batch, stage by stage (module doc), with the
    per-expert work on whole row groups of the oracle's routing (which the
    kernel's routing equals bit for bit)."""
    T, H, I, E, k = d["T"], d["H"], d["I"], d["E"], d["k"]
    ref = W.expert_forward_w8a8(d)
    a = ws_arrays(d, ws)
    # 1. x quantization, bit for bit
    assert np.array_equal(a["xq"], ref["xq"]), f"{what}: x codes"
    assert np.array_equal(a["xs"].view(np.uint32), ref["sx"].view(np.uint32)), f"{what}: x scales"
    rt = ref["routing"]
    off, perm, act = rt["offsets"], rt["perm"], rt["active"]
    w = d["topk_weights"].reshape(-1).astype(np.float64)
    out3 = np.zeros((T, H), dtype=np.float64)
    n_diff = 0
    for e in act[1: 1 + act[0]]:
        e = int(e)
        r0, r1 = int(off[e]), int(off[e + 1])
        slots = perm[r0:r1]
        toks = slots // k
        # 2. h quantization of the expert's rows
        A = W.dequantize_rows_blocks(a["xq"][toks], a["xs"][toks])
        wgu = W._weights_f64(d["w_gate_up"][e], d["w_gate_up_scale"][e])
        g, u = A @ wgu[:I].T, A @ wgu[I:].T
        absA, absW = np.abs(A), np.abs(wgu)
        sg, su = absA @ absW[:I].T, absA @ absW[I:].T
        del A, absA, absW, wgu
        h_bits, tol = h_bounds_rows(g, u, sg, su)
        del g, u, sg, su
        n_diff += check_h_quantization(h_bits, tol, a["hq"][r0:r1], a["hs"][r0:r1],
                                       f"{what} expert {e}")
        # 3. the oracle's down projection and weighted sum of the kernel's h
        wd = W._weights_f64(d["w_down"][e], d["w_down_scale"][e])
        y = W.dequantize_rows_blocks(a["hq"][r0:r1], a["hs"][r0:r1]) @ wd.T
        np.add.at(out3, toks, w[slots][:, None] * y)
    say(f"{what}: h codes equal to the oracle's except {n_diff} of {a['hq'].size}")
    assert n_diff <= 0.01 * a["hq"].size
    check_close(got, out3, f"{what} (down + combine of the kernel's h)")
    # 4. end to end
    err = got - ref["out"]
    rms = np.sqrt((ref["out"] ** 2).mean())
    rel = np.sqrt((err ** 2).mean()) / rms
    say(f"{what}: end to end rms error {rel:.2e} of rms, max {np.abs(err).max() / rms:.2e}")
    assert rel <= TOL


SMALL = [
    # T, H, I, E, k, seed, zipf, mask
    (100, 512, 256, 4, 2, 41, None, 0.0),     # ragged tail: 200 rows over 4 experts
    (300, 768, 384, 8, 4, 42, 1.0, 0.1),      # 6 and 3 K tiles, skew, masked ids
    (37, 256, 128, 3, 3, 43, None, 0.0),      # single K tile on both GEMMs
    (600, 512, 640, 16, 8, 44, 1.2, 0.0),     # many experts, some empty
]


@pytest.mark.parametrize("T,H,I,E,k,seed,zipf,mask", SMALL)
def test_forward_w8a8_small_parity(gpu, T, H, I, E, k, seed, zipf, mask):
    d = synth.make_inputs(T, H, I, E, k, seed, zipf=zipf, wdtype="fp8")
    if mask:
        rng = np.random.default_rng(seed)
        ids = d["topk_ids"].copy()
        m = rng.random(ids.shape) < mask
        ids[m] = -1
        d["topk_ids"] = ids
    say("forward w8a8", T, H, I, E, k, seed)
    got, ws = forward_a8(d)
    check_step(d, got, ws, f"w8a8 T={T} H={H} I={I} E={E} k={k}")


def test_forward_w8a8_bf16_output_and_determinism(gpu):
    d = synth.make_inputs(260, 512, 256, 6, 2, 45, wdtype="fp8")
    say("forward w8a8 determinism")
    a, _ = forward_a8(d)
    b, _ = forward_a8(d)
    assert np.array_equal(a.view(np.uint32), b.view(np.uint32))
    h16, _ = forward_a8(d, torch.bfloat16)
    ref16 = torch.from_numpy(a).to(torch.bfloat16).float().numpy()
    assert np.array_equal(h16, ref16)


def grid_inputs(T, H, I, E, k, seed):
    """Activations whose 128-blocks are e4m3 values times 2^m with amax
    448 * 2^m, and power-of-two weight block scales: every quantization of
    x is exact."""
    d = synth.make_inputs(T, H, I, E, k, seed, wdtype="fp8")
    rng = np.random.default_rng(seed)
    codes = np.array([c for c in range(256) if (c & 0x7F) != 0x7F], dtype=np.uint8)
    vals = O.e4m3fn_to_f32(codes).astype(np.float64)
    x = rng.choice(vals, size=(T, H // 128, 128))
    x[:, :, 0] = 448.0
    x = (x * np.ldexp(1.0, rng.integers(-9, -4, size=(T, H // 128, 1)))).reshape(T, H)
    d["x"] = synth.bf16_bits_from_f32(x.astype(np.float32))
    for key in ("w_gate_up_scale", "w_down_scale"):
        d[key] = np.ldexp(1.0, np.round(np.log2(d[key])).astype(np.int64)).astype(np.float32)
    return d


def test_forward_w8a8_exact_grid(gpu):
    # x quantizes exactly: the GPU's quantized x must reproduce x itself
    d = grid_inputs(T=64, H=256, I=256, E=3, k=2, seed=46)
    say("forward w8a8 exact grid")
    got, ws = forward_a8(d)
    a = ws_arrays(d, ws)
    assert np.array_equal(W.dequantize_rows_blocks(a["xq"], a["xs"]),
                          O.bf16_to_f32(d["x"]).astype(np.float64))
    check_step(d, got, ws, "w8a8 exact grid")


@pytest.mark.timeout(900)
@pytest.mark.parametrize("name", [n for n, w in synth.WORKLOADS.items() if w.act8])
def test_forward_w8a8_workload_all_tokens(gpu, name):
    """The fp8-activation workloads at full size, every token."""
    d = synth.make_workload(name)
    say("forward w8a8 workload", name)
    got, ws = forward_a8(d)
    say("forward w8a8 workload", name, "oracle on all", d["T"], "tokens")
    check_step(d, got, ws, f"workload {name} (all {d['T']} tokens)")


def test_w8a8_shape_limits(gpu):
    assert eaas.eaas_workspace_bytes(8, 384, 128, 2, 1, eaas.EAAS_FP8_E4M3_A8) == 0
    assert eaas.eaas_workspace_bytes(8, 512, 128, 2, 1, eaas.EAAS_FP8_E4M3_A8) > \
        eaas.eaas_workspace_bytes(8, 512, 128, 2, 1, eaas.EAAS_FP8_E4M3)


@pytest.mark.parametrize("case", ["random", "grid"])
def test_fp8_mfma_accumulation_error(gpu, case):
    """The down projection (plain epilogue) of the kernel's own quantized h
    against the exact product: |y - y_exact| <= MFMA_EPS * sum|h w|."""
    if case == "random":
        d = synth.make_inputs(300, 512, 1024, 4, 2, 51, wdtype="fp8")
    else:
        d = grid_inputs(T=64, H=256, I=256, E=3, k=2, seed=46)
    T, H, I, E, k = d["T"], d["H"], d["I"], d["E"], d["k"]
    say("fp8 MFMA accumulation", case, T, H, I, E, k)
    dev = to_device(d)
    A8 = eaas.EAAS_FP8_E4M3_A8
    rt = eaas.alloc_routing(T, k, E)
    ws = eaas.alloc_workspace(T, H, I, E, k, A8)
    eaas.eaas_route_permute(dev["topk_ids"], E, rt, ws, H=H, I=I)
    y = torch.zeros((T * k, H), dtype=torch.float32, device="cuda")
    eaas.eaas_expert_ffn_grouped(dev["x"], rt, dev["w_gate_up"], dev["w_down"], y, ws, k,
                                 dev["w_gate_up_scale"], dev["w_down_scale"], act8=True)
    torch.cuda.synchronize()
    yg = y.cpu().numpy()
    a = ws_arrays(d, ws)
    off = rt["offsets"].cpu().numpy()
    worst = 0.0
    for e in range(E):
        r0, r1 = int(off[e]), int(off[e + 1])
        if r1 <= r0:
            continue
        wd = W._weights_f64(d["w_down"][e], d["w_down_scale"][e])
        hv = W.dequantize_rows_blocks(a["hq"][r0:r1], a["hs"][r0:r1])
        rel = np.abs(yg[r0:r1] - hv @ wd.T) / (np.abs(hv) @ np.abs(wd.T))
        worst = max(worst, float(rel.max()))
    say(f"fp8 MFMA accumulation {case}: worst |dy| / sum|h w| = 2^{np.log2(worst):.1f}")
    assert worst <= MFMA_EPS


def test_forward_w8a8_graph_replay_matches_eager(gpu):
    """The fp8-activation step captured in a graph: every replay, with eager
    work between replays, gives the eager result bit for bit."""
    d = synth.make_inputs(200, 512, 256, 6, 2, 47, wdtype="fp8")
    say("forward w8a8 graph replay")
    dev = to_device(d)
    E, twoI, _ = dev["w_gate_up"].shape
    ws = eaas.alloc_workspace(200, 512, twoI // 2, E, 2, eaas.EAAS_FP8_E4M3_A8)
    out = torch.zeros((200, 512), dtype=torch.float32, device="cuda")

    def step():
        eaas.eaas_expert_forward(dev["x"], dev["topk_ids"], dev["topk_weights"], dev["w_gate_up"],
                                 dev["w_down"], out, ws, dev["w_gate_up_scale"],
                                 dev["w_down_scale"], act8=True)

    step()
    torch.cuda.synchronize()
    ref = out.clone()
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        step()
    torch.cuda.current_stream().wait_stream(s)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        step()
    for _ in range(3):
        out.zero_()
        ws.fill_(0x7F)  # the step must rebuild every intermediate itself
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(out.view(torch.int32), ref.view(torch.int32))
