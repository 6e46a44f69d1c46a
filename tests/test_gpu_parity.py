"""GPU parity of the HIP path (through the C ABI) against the CPU oracle.

Routing must match bit-exactly.  Outputs (fp32 output mode) must satisfy
max|gpu - oracle| <= 2e-2 * RMS(oracle).  Every case prints its name before
touching the GPU.
"""
import json
import os

import numpy as np
import pytest
import torch

from oracle import eaas_oracle as O
from paper_2509_17863_amd import eaas, synth
from paper_2509_17863_amd.device_io import bf16_tensor_to_bits, to_device

pytestmark = pytest.mark.gpu

TOL = 2e-2
GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
ROUTE_KEYS = ("counts", "offsets", "perm", "inv", "active")


def say(*a):
    print("[gpu-case]", *a, flush=True)


def gpu_route(ids_np, E, H=128, I=128):
    T, k = ids_np.shape
    ids = torch.from_numpy(np.ascontiguousarray(ids_np, dtype=np.int32)).cuda()
    r = eaas.alloc_routing(T, k, E)
    ws = eaas.alloc_workspace(T, H, I, E, k)
    eaas.eaas_route_permute(ids, E, r, ws, H=H, I=I)
    torch.cuda.synchronize()
    return {key: v.cpu().numpy() for key, v in r.items()}


def assert_routing_equal(got, ref, R, E):
    assert np.array_equal(got["counts"][:E], ref["counts"])
    assert np.array_equal(got["offsets"][:E + 1], ref["offsets"])
    assert np.array_equal(got["perm"][:R], ref["perm"])
    assert np.array_equal(got["inv"][:R], ref["inv"])
    assert np.array_equal(got["active"][:E + 1], ref["active"])


def forward(dev, k, out_dtype=torch.float32, routing=None, out=None, stream=None):
    T, H = dev["x"].shape
    E, twoI, _ = dev["w_gate_up"].shape
    wdt = eaas.EAAS_FP8_E4M3 if dev["w_gate_up"].element_size() == 1 else eaas.EAAS_BF16
    ws = eaas.alloc_workspace(T, H, twoI // 2, E, k, wdt)
    if out is None:
        out = torch.full((T, H), float("nan"), dtype=out_dtype, device="cuda")
    eaas.eaas_expert_forward(dev["x"], dev["topk_ids"], dev["topk_weights"], dev["w_gate_up"],
                             dev["w_down"], out, ws, dev["w_gate_up_scale"],
                             dev["w_down_scale"], routing=routing, stream=stream)
    return out


def check_close(got, ref, what):
    got = np.asarray(got, dtype=np.float64)
    rms = float(np.sqrt((ref ** 2).mean())) if ref.size else 0.0
    err = float(np.abs(got - ref).max()) if ref.size else 0.0
    say(f"{what}: max_abs_err={err:.3e} rms={rms:.3e} ratio={err / max(rms, 1e-30):.2e}")
    assert np.isfinite(got).all(), f"{what}: non-finite output"
    assert err <= TOL * rms, f"{what}: {err} > {TOL} * {rms}"


# ---------------------------------------------------------------- routing
def test_route_hand_fixtures(gpu):
    cases = json.load(open(os.path.join(GOLDEN, "routing_hand.json")))["cases"]
    for c in cases:
        ids = np.array(c["topk_ids"], np.int32)
        say("route hand", ids.shape, c["E"])
        got = gpu_route(ids, c["E"])
        for key in ROUTE_KEYS:
            assert got[key][: len(c[key])].tolist() == c[key], key


ROUTE_CASES = [
    # (T, E, k, mask fraction, seed)
    (1, 1, 1, 0.0, 0), (3, 8, 2, 0.0, 1), (100, 8, 2, 0.3, 2), (1000, 3, 8, 0.1, 3),
    (2047, 64, 1, 0.0, 4), (2049, 128, 8, 0.05, 5), (513, 1024, 4, 0.0, 6),
    (5000, 1024, 2, 0.5, 7), (300, 5, 5, 0.0, 8),
    # around the single-workgroup path's limit of 8192 slots
    (1024, 16, 4, 0.2, 9), (8192, 1024, 1, 0.1, 10), (8193, 7, 1, 0.0, 11), (1, 1024, 8, 0.5, 12),
    (4096, 8, 2, 0.0, 13),
    # the largest k (64): many slots per token
    (50, 32, 64, 0.1, 14), (129, 1024, 64, 0.0, 15),
]


@pytest.mark.parametrize("T,E,k,mask,seed", ROUTE_CASES)
def test_route_random_bitexact(gpu, T, E, k, mask, seed):
    rng = np.random.default_rng(seed)
    ids = rng.integers(0, E, size=(T, k)).astype(np.int32)
    if mask:
        m = rng.random(ids.shape) < mask
        ids[m] = rng.choice(np.array([-1, E, -7, 1 << 20], np.int32), size=int(m.sum()))
    say("route random", T, E, k, mask)
    assert_routing_equal(gpu_route(ids, E), O.route_permute(ids, E), T * k, E)


def test_route_all_on_one_expert_and_empty(gpu):
    ids = np.full((3000, 4), 6, np.int32)
    say("route one expert")
    assert_routing_equal(gpu_route(ids, 9), O.route_permute(ids, 9), 12000, 9)
    ids = np.full((70, 2), -1, np.int32)
    say("route all masked")
    assert_routing_equal(gpu_route(ids, 4), O.route_permute(ids, 4), 140, 4)


@pytest.mark.parametrize("name", list(synth.WORKLOADS))
def test_route_workloads_bitexact(gpu, name):
    d = synth.make_workload(name, weights=False)
    say("route workload", name)
    got = gpu_route(d["topk_ids"], d["E"], d["H"], d["I"])
    assert_routing_equal(got, O.route_permute(d["topk_ids"], d["E"]), d["T"] * d["k"], d["E"])


# ---------------------------------------------------------------- forward, small
SMALL = [
    # T, H, I, E, k, seed, zipf, wdtype, mask
    (64, 256, 128, 8, 2, 0, None, "bf16", 0.0),      # the tiny workload's shape
    (300, 384, 256, 6, 2, 21, None, "bf16", 0.0),    # ragged tails, N not a multiple of 256
    (700, 512, 384, 5, 3, 22, 2.0, "bf16", 0.1),     # several M tiles, skew, masked slots
    (97, 256, 256, 40, 4, 23, 1.5, "bf16", 0.0),     # many small experts, some empty
    (1, 256, 128, 4, 2, 24, None, "bf16", 0.0),      # single token
    (130, 512, 256, 4, 3, 25, None, "fp8", 0.0),     # fp8 block-scaled weights
    (600, 768, 512, 3, 2, 26, None, "fp8", 0.2),     # fp8, several tiles, masked
    (200, 384, 384, 5, 2, 27, 1.5, "fp8", 0.1),      # fp8, gate/up N = 768, down N = 384
    (40, 256, 128, 80, 64, 28, None, "bf16", 0.05),  # the largest k: 64 slots per token
    (24, 512, 256, 72, 64, 29, 1.2, "fp8", 0.0),     # the largest k, fp8 weights
]


@pytest.mark.parametrize("T,H,I,E,k,seed,zipf,wdtype,mask", SMALL)
def test_forward_small_parity(gpu, T, H, I, E, k, seed, zipf, wdtype, mask):
    d = synth.make_inputs(T, H, I, E, k, seed, zipf=zipf, wdtype=wdtype)
    if mask:
        rng = np.random.default_rng(seed)
        ids = d["topk_ids"].copy()
        ids[rng.random(ids.shape) < mask] = -1
        d["topk_ids"] = ids
    ref = O.expert_forward(d)
    dev = to_device(d)
    say("forward small", T, H, I, E, k, wdtype, mask)
    r = eaas.alloc_routing(T, k, E)
    out = forward(dev, k, routing=r)
    torch.cuda.synchronize()
    got_r = {key: v.cpu().numpy() for key, v in r.items()}
    assert_routing_equal(got_r, ref["routing"], T * k, E)
    check_close(out.cpu().numpy(), ref["out"], f"small {T}x{H}x{I} E{E} k{k} {wdtype}")


def test_forward_hand_fixture(gpu):
    # the hand-worked FFN fixture embedded in a 128-aligned shape (zero padding)
    c = json.load(open(os.path.join(GOLDEN, "ffn_hand.json")))
    H, I, E = 128, 128, 2
    x = np.zeros((1, H), np.float32)
    x[0, :2] = c["x"][0]
    wgu = np.zeros((E, 2 * I, H), np.float32)
    wd = np.zeros((E, H, I), np.float32)
    for e in range(E):
        wgu[e, 0, :2] = c["w_gate_up"][e][0]
        wgu[e, I, :2] = c["w_gate_up"][e][1]
        wd[e, :2, 0] = [row[0] for row in c["w_down"][e]]
    d = dict(T=1, H=H, I=I, E=E, k=2, wdtype="bf16", x=synth.bf16_bits_from_f32(x),
             topk_ids=np.array(c["topk_ids"], np.int32),
             topk_weights=np.array(c["topk_weights"], np.float32),
             w_gate_up=synth.bf16_bits_from_f32(wgu), w_down=synth.bf16_bits_from_f32(wd),
             w_gate_up_scale=None, w_down_scale=None)
    say("forward hand fixture")
    out = forward(to_device(d), 2).cpu().numpy()
    assert np.array_equal(out[0, :2], np.array(c["out"][0], np.float32))
    assert np.all(out[0, 2:] == 0)


# ---------------------------------------------------------------- forward, full size
def oracle_out_all_tokens(d, chunk=2048):
    """The oracle's fp64 output for every token of a full-size batch, computed
    over sub-batches of `chunk` tokens (a token's outputs depend on that token
    alone) with each expert's weights converted to fp64 once."""
    E, T = d["E"], d["T"]
    w64 = ([], [])
    for e in range(E):
        wg, wu, wd = O.expert_weights_f64(d, e)
        w64[0].append(np.concatenate([wg, wu]))
        w64[1].append(wd)
    out = np.empty((T, d["H"]), dtype=np.float64)
    for a in range(0, T, chunk):
        b = min(T, a + chunk)
        out[a:b] = O.expert_forward(O.sub_batch(d, np.arange(a, b)), weights=w64)["out"]
    return out


@pytest.mark.timeout(900)
@pytest.mark.parametrize("name", list(synth.WORKLOADS))
def test_forward_workload_all_tokens(gpu, name):
    """Every token of every full-size workload against the oracle (fp32
    output), plus determinism and the bf16 output being RNE of the fp32 one."""
    if synth.WORKLOADS[name].act8:
        pytest.skip("fp8-activation workloads: tests/test_gpu_w8a8.py (all tokens there too)")
    d = synth.make_workload(name)
    T, k = d["T"], d["k"]
    dev = to_device(d)
    say("forward workload", name)
    out32 = forward(dev, k, torch.float32)
    out16 = forward(dev, k, torch.bfloat16)
    again = forward(dev, k, torch.float32)
    torch.cuda.synchronize()
    o32 = out32.cpu().numpy()
    # determinism: bitwise identical reruns
    assert np.array_equal(o32.view(np.uint32), again.cpu().numpy().view(np.uint32))
    # bf16 output is round-to-nearest-even of the fp32 result
    ref16 = torch.from_numpy(o32).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(bf16_tensor_to_bits(out16), ref16)
    assert np.isfinite(o32).all()
    del dev, out32, out16, again
    say("forward workload", name, "oracle on all", T, "tokens")
    ref = oracle_out_all_tokens(d)
    check_close(o32, ref, f"workload {name} (all {T} tokens)")


# ------------------------------------------------- exact h stage (integer data)
def integer_bits(rng, shape, p, fp8=False):
    """Entries -1, 0, +1 with P(nonzero) = p, as bf16 (or e4m3fn) bits: exact
    in either format, and every fp32 sum of them is exact."""
    u = rng.random(shape, dtype=np.float32)
    if fp8:
        one, neg = np.uint8(0x38), np.uint8(0xB8)       # e4m3fn +1.0, -1.0
        return np.where(u < p / 2, neg, np.where(u < p, one, np.uint8(0)))
    one, neg = np.uint16(0x3F80), np.uint16(0xBF80)     # bf16 +1.0, -1.0
    return np.where(u < p / 2, neg, np.where(u < p, one, np.uint16(0)))


def integer_workload(name, seed=77):
    """The workload's batch and routing with x and weights replaced by
    sparse integers (fp8 weights keep scales of exactly 1): G and U are then
    integers below 2^24, exact in any fp32 summation order.  The density
    gives G a standard deviation near 8, across the curved part of silu."""
    d = synth.make_workload(name, weights=False)
    T, H, I, E = d["T"], d["H"], d["I"], d["E"]
    fp8 = synth.WORKLOADS[name].wdtype == "fp8"
    rng = np.random.default_rng(seed)
    p = float(np.sqrt(64.0 / H))
    d["x"] = integer_bits(rng, (T, H), p)
    d["w_gate_up"] = np.stack([integer_bits(rng, (2 * I, H), p, fp8) for _ in range(E)])
    d["w_down"] = np.stack([integer_bits(rng, (H, I), np.sqrt(64.0 / I), fp8) for _ in range(E)])
    d["w_gate_up_scale"] = np.ones((E, 2 * I // 128, H // 128), np.float32) if fp8 else None
    d["w_down_scale"] = np.ones((E, H // 128, I // 128), np.float32) if fp8 else None
    d["wdtype"] = "fp8" if fp8 else "bf16"
    return d


# The kernel evaluates silu(g) * u with the hardware exp and reciprocal: for
# |g| <= 88 its fp32 value lies within 2^-17 (relative) of the exact one.
# Where [v (1 - 2^-16), v (1 + 2^-16)] holds a bf16 rounding boundary either
# rounding is accepted; everywhere else h must match exactly.
H_REL = 2.0 ** -16


def exact_h_candidates(g, u):
    """bf16 values h may take for exact integer g, u (fp64 arrays)."""
    with np.errstate(over="ignore"):
        v = g / (1.0 + np.exp(-g)) * u
    lo = O.bf16_to_f32(O.f32_to_bf16_rne((v * (1 - H_REL)).astype(np.float32)))
    hi = O.bf16_to_f32(O.f32_to_bf16_rne((v * (1 + H_REL)).astype(np.float32)))
    return lo, hi


@pytest.mark.timeout(900)
@pytest.mark.parametrize("name", ["mixtral", "qwen3", "dsv3_prefill", "dsv3_decode"])
def test_gate_up_h_exact_on_integer_data(gpu, name):
    """Full-size gate/up stage with integer x and weights: every h of the
    grouped layout equals the exactly computed value's bf16 rounding (either
    neighbour only where the exact value is within 2^-16 of a rounding
    boundary).  An indexing slip anywhere in the grouped GEMM (a wrong row,
    column, expert or K tile) moves G by whole integers and fails here."""
    d = integer_workload(name)
    T, H, I, E, k = d["T"], d["H"], d["I"], d["E"], d["k"]
    wdt = eaas.EAAS_FP8_E4M3 if d["wdtype"] == "fp8" else eaas.EAAS_BF16
    dev = to_device(d)
    say("exact h", name, d["wdtype"])
    ws = eaas.alloc_workspace(T, H, I, E, k, wdt)
    out = torch.empty((T, H), dtype=torch.float32, device="cuda")
    eaas.eaas_expert_forward(dev["x"], dev["topk_ids"], dev["topk_weights"], dev["w_gate_up"],
                             dev["w_down"], out, ws, dev["w_gate_up_scale"], dev["w_down_scale"])
    torch.cuda.synchronize()
    h = eaas.workspace_view(ws, T, H, I, E, k, wdt, eaas.EAAS_WS_H).cpu().numpy().view(np.uint16)
    h = O.bf16_to_f32(h.reshape(T * k, I))
    del dev, ws, out
    rt = O.route_permute(d["topk_ids"], E)
    off, perm = rt["offsets"], rt["perm"]
    x = O.bf16_to_f32(d["x"])
    n_amb = n_all = 0
    for e in range(E):
        r0, r1 = int(off[e]), int(off[e + 1])
        if r1 == r0:
            continue
        if d["wdtype"] == "fp8":
            wgu = O.e4m3fn_to_f32(d["w_gate_up"][e])
        else:
            wgu = O.bf16_to_f32(d["w_gate_up"][e])
        a = x[perm[r0:r1] // k]
        g = (a @ wgu[:I].T).astype(np.float64)   # integers < 2^24: exact in fp32
        u = (a @ wgu[I:].T).astype(np.float64)
        # (below -88 the kernel's exp overflows to a silu of 0: the data
        # never reach it, g has a standard deviation near 8)
        assert np.abs(g).max() < 2 ** 24 and g.min() > -80
        lo, hi = exact_h_candidates(g, u)
        got = h[r0:r1]
        ok = (got == lo) | (got == hi)
        bad = np.argwhere(~ok)
        assert bad.size == 0, (f"expert {e}: {len(bad)} h values wrong, first (row, col) "
                               f"{bad[:4].tolist()}: got {got[tuple(bad[0])]}, "
                               f"want {lo[tuple(bad[0])]} or {hi[tuple(bad[0])]}")
        n_amb += int((lo != hi).sum())
        n_all += lo.size
    say(f"exact h {name}: {n_all} values equal; {n_amb} near a rounding boundary "
        f"({n_amb / max(n_all, 1):.2e})")
    assert n_all == T * k * I


# ---------------------------------------------------------------- properties
def _mid_inputs(wdtype="bf16", seed=31):
    return synth.make_inputs(700, 512, 256, 8, 4, seed, zipf=1.0, wdtype=wdtype)


def test_modular_equals_fused_bitwise(gpu):
    d = _mid_inputs()
    dev = to_device(d)
    T, H, I, E, k = d["T"], d["H"], d["I"], d["E"], d["k"]
    say("modular vs fused")
    fused = forward(dev, k, torch.float32)
    r = eaas.alloc_routing(T, k, E)
    ws = eaas.alloc_workspace(T, H, I, E, k)
    eaas.eaas_route_permute(dev["topk_ids"], E, r, ws, H=H, I=I)
    y = torch.empty((T * k, H), dtype=torch.float32, device="cuda")
    eaas.eaas_expert_ffn_grouped(dev["x"], r, dev["w_gate_up"], dev["w_down"], y, ws, k)
    out = torch.empty((T, H), dtype=torch.float32, device="cuda")
    eaas.eaas_unpermute_combine(y, r, dev["topk_weights"], out, E, I=I)
    torch.cuda.synchronize()
    assert np.array_equal(fused.cpu().numpy().view(np.uint32), out.cpu().numpy().view(np.uint32))
    # the unweighted per-row expert outputs against the oracle
    ref = O.expert_forward(d)
    check_close(y.cpu().numpy(), ref["y"], "y_perm rows")


def test_in_place_write_back(gpu):
    d = _mid_inputs(seed=32)
    dev = to_device(d)
    k = d["k"]
    say("in place")
    ref = forward(dev, k, torch.bfloat16)
    x2 = dev["x"].clone()
    dev2 = dict(dev, x=x2)
    forward(dev2, k, out=x2)
    torch.cuda.synchronize()
    assert np.array_equal(bf16_tensor_to_bits(x2), bf16_tensor_to_bits(ref))


def test_token_permutation_equivariance_bitwise(gpu):
    d = _mid_inputs(seed=33)
    p = np.random.default_rng(3).permutation(d["T"])
    say("equivariance")
    a = forward(to_device(d), d["k"]).cpu().numpy()
    b = forward(to_device(O.sub_batch(d, p)), d["k"]).cpu().numpy()
    assert np.array_equal(a[p].view(np.uint32), b.view(np.uint32))


@pytest.mark.parametrize("wdtype", ["bf16", "fp8"])
def test_batch_split_invariance_bitwise(gpu, wdtype):
    """A token's output does not depend on the batch around it: the first
    64 tokens alone (a decode-sized batch: at most one M tile per expert,
    nontemporal weight reads for bf16) give the same bits as inside the
    whole 4096-token batch (several M tiles per expert, default reads), and
    so does a 300-token slice from the middle."""
    d = synth.make_inputs(4096, 512, 256, 8, 2, 34, zipf=1.1, wdtype=wdtype)
    say("batch split", wdtype)
    whole = forward(to_device(d), d["k"]).cpu().numpy()
    for lo, hi in ((0, 64), (1800, 2100)):
        part = forward(to_device(O.sub_batch(d, np.arange(lo, hi))), d["k"]).cpu().numpy()
        assert np.array_equal(part.view(np.uint32), whole[lo:hi].view(np.uint32)), (lo, hi)


def test_graph_replay_matches_eager(gpu):
    d = _mid_inputs(seed=34)
    dev = to_device(d)
    T, H, I, E, k = d["T"], d["H"], d["I"], d["E"], d["k"]
    say("graph replay")
    eager = forward(dev, k).cpu().numpy()
    ws = eaas.alloc_workspace(T, H, I, E, k)
    out = torch.empty((T, H), dtype=torch.float32, device="cuda")
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        eaas.eaas_expert_forward(dev["x"], dev["topk_ids"], dev["topk_weights"],
                                 dev["w_gate_up"], dev["w_down"], out, ws)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        eaas.eaas_expert_forward(dev["x"], dev["topk_ids"], dev["topk_weights"],
                                 dev["w_gate_up"], dev["w_down"], out, ws)
    for i in range(3):
        out.fill_(float("nan"))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert np.array_equal(out.cpu().numpy().view(np.uint32), eager.view(np.uint32)), i


def test_concurrent_streams_are_independent(gpu):
    """The library keeps no state between calls: two forwards of different
    batches in flight at once on two streams (own workspaces) give the
    results each gives alone, bit for bit."""
    da = _mid_inputs(seed=36)
    db = synth.make_inputs(300, 512, 256, 8, 4, 37, zipf=None, wdtype="fp8")
    deva, devb = to_device(da), to_device(db)
    say("concurrent streams")
    alone_a = forward(deva, da["k"]).cpu().numpy()
    alone_b = forward(devb, db["k"]).cpu().numpy()
    torch.cuda.synchronize()
    sa, sb = torch.cuda.Stream(), torch.cuda.Stream()
    outs = []
    for _ in range(3):
        oa = torch.full((da["T"], da["H"]), float("nan"), device="cuda")
        ob = torch.full((db["T"], db["H"]), float("nan"), device="cuda")
        sa.wait_stream(torch.cuda.current_stream())
        sb.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(sa):
            forward(deva, da["k"], out=oa, stream=sa.cuda_stream)
        with torch.cuda.stream(sb):
            forward(devb, db["k"], out=ob, stream=sb.cuda_stream)
        outs.append((oa, ob))
    torch.cuda.synchronize()
    for oa, ob in outs:
        assert np.array_equal(oa.cpu().numpy().view(np.uint32), alone_a.view(np.uint32))
        assert np.array_equal(ob.cpu().numpy().view(np.uint32), alone_b.view(np.uint32))


def test_forward_1024_experts(gpu):
    """The largest expert count the scheduler takes (1024): mostly one- to
    three-row experts, several empty."""
    d = synth.make_inputs(300, 128, 128, 1024, 8, 38, zipf=None, wdtype="bf16")
    ref = O.expert_forward(d)
    say("forward E=1024")
    dev = to_device(d)
    r = eaas.alloc_routing(d["T"], d["k"], d["E"])
    got = forward(dev, d["k"], routing=r).cpu().numpy()
    assert_routing_equal({key: v.cpu().numpy() for key, v in r.items()}, ref["routing"],
                         d["T"] * d["k"], d["E"])
    check_close(got, ref["out"], "E=1024")


TILE_EDGE_COUNTS = [1, 31, 32, 33, 63, 64, 65, 95, 96, 97, 127, 128, 129, 255, 256, 257, 0]


@pytest.mark.parametrize("wdtype", ["bf16", "fp8"])
@pytest.mark.parametrize("H,extra", [(128, 0), (384, 0), (256, 3000)])
def test_forward_tile_row_boundaries(gpu, wdtype, H, extra):
    """Experts holding one row less than, exactly, and one row more than a
    32-row block, a 96-row fp8 tile, a half (128-row) and a whole (256-row)
    bf16 tile.  Without `extra` the batch is decode-sized (R <= 256 E: the
    small-tile weight ring and the nontemporal weight reads); an extra expert
    with `extra` rows makes it prefill-sized.  K = H gives 2, 6 and 4 K tiles."""
    counts = TILE_EDGE_COUNTS + ([extra] if extra else [])
    E, T, I = len(counts), int(sum(counts)), 128
    rng = np.random.default_rng(40 + H + extra)
    d = synth.make_inputs(T, H, I, E, 1, 41, zipf=None, wdtype=wdtype)
    ids = np.repeat(np.arange(E, dtype=np.int32), counts)
    d["topk_ids"] = rng.permutation(ids).reshape(T, 1).astype(np.int32)
    d["topk_weights"] = np.ones((T, 1), dtype=np.float32)
    say(f"tile edges {wdtype} H={H} extra={extra} T={T} E={E}")
    ref = O.expert_forward(d)
    assert np.array_equal(ref["routing"]["counts"], np.asarray(counts))
    dev = to_device(d)
    r = eaas.alloc_routing(T, 1, E)
    got = forward(dev, 1, routing=r).cpu().numpy()
    assert_routing_equal({key: v.cpu().numpy() for key, v in r.items()}, ref["routing"], T, E)
    check_close(got, ref["out"], f"tile edges {wdtype} H={H}")


@pytest.mark.parametrize("wdtype", ["bf16", "fp8", "a8"])
def test_forward_at_the_32bit_offset_limit(gpu, wdtype):
    """The largest batch the 32-bit element offsets allow at H = 1024:
    T*H = 2^31 - 1024 (x is 4 GiB, so the DMA's byte offsets into it reach
    2^32 - 2048).  Routing against a stable sort on every slot; the output of
    the first, middle and last tokens against the oracle (fp8 activations:
    its RMS error, as for the random shapes)."""
    from oracle import w8a8_oracle as W

    T, H, I, E, k = (1 << 21) - 1, 1024, 128, 4, 2
    act8 = wdtype == "a8"
    say(f"offset limit {wdtype} T={T} H={H}")
    dw = synth.make_inputs(1, H, I, E, k, 44, wdtype="bf16" if wdtype == "bf16" else "fp8")
    g = torch.Generator(device="cuda").manual_seed(45)
    x = torch.randn(T, H, generator=g, device="cuda").to(torch.bfloat16)
    e0 = torch.randint(0, E, (T,), generator=g, device="cuda")
    e1 = (e0 + torch.randint(1, E, (T,), generator=g, device="cuda")) % E
    ids = torch.stack([e0, e1], 1).to(torch.int32).contiguous()
    w = torch.rand(T, k, generator=g, device="cuda") + 0.1
    w = (w / w.sum(1, keepdim=True)).contiguous()
    dev = dict(to_device(dw), x=x, topk_ids=ids, topk_weights=w)
    r = eaas.alloc_routing(T, k, E)
    if act8:
        ws = eaas.alloc_workspace(T, H, I, E, k, eaas.EAAS_FP8_E4M3_A8)
        out = torch.full((T, H), float("nan"), dtype=torch.float32, device="cuda")
        eaas.eaas_expert_forward(x, ids, w, dev["w_gate_up"], dev["w_down"], out, ws,
                                 dev["w_gate_up_scale"], dev["w_down_scale"], routing=r,
                                 act8=True)
        del ws
    else:
        out = forward(dev, k, routing=r)
    torch.cuda.synchronize()
    flat = ids.flatten().to(torch.int64)
    assert torch.equal(r["counts"][:E].to(torch.int64), torch.bincount(flat, minlength=E))
    assert torch.equal(r["perm"][:T * k].to(torch.int64), torch.argsort(flat, stable=True))
    idx = np.r_[0:16, T // 2 - 8:T // 2 + 8, T - 32:T]
    ti = torch.from_numpy(idx).cuda()
    ds = dict(dw, T=len(idx), x=bf16_tensor_to_bits(x[ti]), topk_ids=ids[ti].cpu().numpy(),
              topk_weights=w[ti].cpu().numpy())
    got = out[ti].cpu().numpy()
    del out, x, dev, r
    torch.cuda.empty_cache()
    if act8:
        ref = W.expert_forward_w8a8(ds)["out"]
        rms = float(np.sqrt((ref ** 2).mean()))
        err = float(np.sqrt(((got.astype(np.float64) - ref) ** 2).mean()))
        say(f"offset limit a8: rms_err={err:.3e} rms={rms:.3e}")
        assert np.isfinite(got).all() and err <= TOL * rms
    else:
        check_close(got, O.expert_forward(ds)["out"], f"offset limit {wdtype}")


def test_fp8_path_matches_bf16_on_representable_weights(gpu):
    d8 = synth.make_inputs(300, 512, 256, 4, 2, 35, wdtype="fp8")
    wgu, wdn = O.weights_f32(d8)
    # weights q*s are bf16-representable when the scales are powers of two
    for key in ("w_gate_up_scale", "w_down_scale"):
        d8[key] = np.exp2(np.round(np.log2(d8[key]))).astype(np.float32)
    wgu, wdn = O.weights_f32(d8)
    db = dict(d8, wdtype="bf16", w_gate_up=synth.bf16_bits_from_f32(wgu),
              w_down=synth.bf16_bits_from_f32(wdn), w_gate_up_scale=None, w_down_scale=None)
    assert np.array_equal(O.bf16_to_f32(db["w_gate_up"]), wgu)
    say("fp8 vs bf16")
    a = forward(to_device(d8), 2).cpu().numpy().astype(np.float64)
    b = forward(to_device(db), 2).cpu().numpy().astype(np.float64)
    rms = np.sqrt((b ** 2).mean())
    # equal up to fp32 accumulation order (and the rare bf16 flip of h it causes);
    # a wrong fp8 decode or scale index would be off by O(rms)
    assert np.abs(a - b).max() <= 2e-3 * rms


def test_empty_batch_is_noop(gpu):
    say("empty batch")
    x = torch.empty((0, 256), dtype=torch.bfloat16, device="cuda")
    ids = torch.empty((0, 2), dtype=torch.int32, device="cuda")
    w = torch.empty((0, 2), dtype=torch.float32, device="cuda")
    wgu = torch.zeros((4, 256, 256), dtype=torch.bfloat16, device="cuda")
    wd = torch.zeros((4, 256, 128), dtype=torch.bfloat16, device="cuda")
    out = torch.empty((0, 256), dtype=torch.float32, device="cuda")
    ws = torch.empty(256, dtype=torch.uint8, device="cuda")
    eaas.eaas_expert_forward(x, ids, w, wgu, wd, out, ws)
    torch.cuda.synchronize()


# ------------------------------------------- poisoned workspace, output canaries
CANARY_F32 = np.uint32(0x7FA5A5A5)   # a NaN payload no kernel writes


@pytest.mark.parametrize("wdtype", ["bf16", "fp8"])
def test_poisoned_workspace_and_canaries(gpu, wdtype):
    """The step rebuilds every intermediate itself: a workspace filled with
    NaN bytes (-1 as int32) gives the clean run's result bit for bit.  Rows
    of guard memory around the output and bytes past the workspace the call
    was given keep their canary values."""
    d = synth.make_inputs(700, 512, 384, 7, 3, 81, zipf=1.3, wdtype=wdtype)
    d["topk_ids"][::11, 1] = -1
    T, H, I, E, k = d["T"], d["H"], d["I"], d["E"], d["k"]
    wdt = eaas.EAAS_FP8_E4M3 if wdtype == "fp8" else eaas.EAAS_BF16
    dev = to_device(d)
    say("poisoned workspace", wdtype)
    clean = forward(dev, k).cpu().numpy()
    n = eaas.eaas_workspace_bytes(T, H, I, E, k, wdt)
    G = 8
    ws_big = torch.full((n + 4096,), 0xFF, dtype=torch.uint8, device="cuda")
    ws_big[n:] = 0xA5
    guard = torch.from_numpy(np.full((T + 2 * G, H), CANARY_F32, np.uint32)).cuda()
    out = guard.view(torch.float32)[G:G + T]
    assert out.is_contiguous()
    eaas.eaas_expert_forward(dev["x"], dev["topk_ids"], dev["topk_weights"], dev["w_gate_up"],
                             dev["w_down"], out, ws_big[:n], dev["w_gate_up_scale"],
                             dev["w_down_scale"])
    torch.cuda.synchronize()
    g = guard.cpu().numpy()
    assert np.all(g[:G] == CANARY_F32) and np.all(g[G + T:] == CANARY_F32), "output guard rows"
    assert np.array_equal(g[G:G + T], clean.view(np.uint32)), "poisoned workspace changed the result"
    assert torch.all(ws_big[n:] == 0xA5).item(), "bytes past the workspace were written"
    # the modular entry points with workspaces of exactly their own size
    nr = eaas.eaas_workspace_bytes_for(T, H, I, E, k, wdt, eaas.EAAS_ENTRY_ROUTE_PERMUTE)
    nf = eaas.eaas_workspace_bytes_for(T, H, I, E, k, wdt, eaas.EAAS_ENTRY_FFN_GROUPED)
    ws_r = torch.full((nr + 256,), 0xA5, dtype=torch.uint8, device="cuda")
    ws_f = torch.full((nf + 256,), 0xFF, dtype=torch.uint8, device="cuda")
    ws_f[nf:] = 0xA5
    r = eaas.alloc_routing(T, k, E)
    eaas.eaas_route_permute(dev["topk_ids"], E, r, ws_r[:nr], H=H, I=I)
    yg = torch.from_numpy(np.full((T * k + 2 * G, H), CANARY_F32, np.uint32)).cuda()
    y = yg.view(torch.float32)[G:G + T * k]
    eaas.eaas_expert_ffn_grouped(dev["x"], r, dev["w_gate_up"], dev["w_down"], y, ws_f[:nf], k,
                                 dev["w_gate_up_scale"], dev["w_down_scale"])
    out2 = torch.empty((T, H), dtype=torch.float32, device="cuda")
    eaas.eaas_unpermute_combine(y, r, dev["topk_weights"], out2, E, I=I)
    torch.cuda.synchronize()
    assert torch.all(ws_r[nr:] == 0xA5).item() and torch.all(ws_f[nf:] == 0xA5).item()
    ygn = yg.cpu().numpy()
    R_valid = int((d["topk_ids"] >= 0).sum())
    assert np.all(ygn[:G] == CANARY_F32) and np.all(ygn[G + T * k:] == CANARY_F32)
    # rows past the valid slots are left untouched
    assert np.all(ygn[G + R_valid:G + T * k] == CANARY_F32)
    assert np.array_equal(out2.cpu().numpy().view(np.uint32), clean.view(np.uint32))


def test_forward_k_above_E(gpu):
    """A server with fewer experts than a token has slots: the slots naming
    other servers' experts are skipped, duplicate ids count twice."""
    rng = np.random.default_rng(82)
    d = synth.make_inputs(300, 256, 256, 3, 2, 82, wdtype="bf16")
    T, E, k = d["T"], d["E"], 8
    extra = rng.choice(np.array([-1, 3, 9], np.int32), size=(T, k - 2))
    extra = np.where(rng.random((T, k - 2)) < 0.3, d["topk_ids"][:, :1], extra).astype(np.int32)
    d["topk_ids"] = np.ascontiguousarray(np.concatenate([d["topk_ids"], extra], 1))
    d["topk_weights"] = np.ascontiguousarray(np.concatenate(
        [d["topk_weights"], rng.random((T, k - 2)).astype(np.float32)], 1))
    d["k"] = k
    ref = O.expert_forward(d)
    say("forward k > E")
    r = eaas.alloc_routing(T, k, E)
    out = forward(to_device(d), k, routing=r)
    torch.cuda.synchronize()
    assert_routing_equal({key: v.cpu().numpy() for key, v in r.items()}, ref["routing"], T * k, E)
    check_close(out.cpu().numpy(), ref["out"], "k=8 > E=3")


@pytest.mark.parametrize("shape", [(300, 256, 256, 1024, 8, 83, None, "bf16"),
                                   (700, 512, 384, 40, 4, 84, 1.5, "bf16"),
                                   (200, 512, 256, 12, 4, 85, 1.2, "fp8")])
def test_scheduler_builds_agree_bitwise(gpu, shape):
    """The two other builds of the GEMM tile scheduler (all E experts
    scanned; every workgroup walking the E experts) find the same tiles:
    bitwise the same output as the library (group-shrink ablation builds)."""
    from paper_2509_17863_amd import _build

    T, H, I, E, k, seed, zipf, wdtype = shape
    d = synth.make_inputs(T, H, I, E, k, seed, zipf=zipf, wdtype=wdtype)
    dev = to_device(d)
    say("scheduler builds", shape)
    ref = forward(dev, k).cpu().numpy()
    try:
        for name in _build.SCHEDULER_VARIANTS:
            eaas.use_library(_build.variant_library(name))
            got = forward(dev, k).cpu().numpy()
            assert np.array_equal(got.view(np.uint32), ref.view(np.uint32)), name
    finally:
        eaas.use_library(None)
