"""GPU parity of the dynamic-batch entry point (several clients' requests,
token counts read on the device, EaaS §3.3 and Algorithm 1 of §4).

Every request's rows must equal, bit for bit, what eaas_expert_forward
writes for those tokens when the requests are concatenated in slot order
(the per-token computation does not depend on the batch around it), and stay
within 2e-2 * RMS of the oracle's segmented step.  Rows past a request's
count, and requests past the capacity, must be left untouched.  Every case
prints its name before touching the GPU.
"""
import numpy as np
import pytest
import torch

from oracle import eaas_oracle as O
from oracle import segments_oracle as S
from paper_2509_17863_amd import eaas, synth
from paper_2509_17863_amd.device_io import bf16_tensor_to_bits, to_device

pytestmark = pytest.mark.gpu

TOL = 2e-2


def say(*a):
    print("[gpu-case]", *a, flush=True)


def make_requests(sizes, H=512, I=256, E=8, k=4, seed=41, wdtype="bf16", pad=5):
    """Requests cut from one seeded batch; each payload buffer holds `pad`
    more rows than its request (garbage rows the server must not read)."""
    T = max(sum(sizes), 1)
    d = synth.make_inputs(T, H, I, E, k, seed, wdtype=wdtype)
    rng = np.random.default_rng(seed + 7)
    reqs, p = [], 0
    for n in sizes:
        cap = n + pad
        x = synth.bf16_bits_from_f32(rng.standard_normal((cap, H)).astype(np.float32))
        ids = rng.integers(-3, E + 3, size=(cap, k)).astype(np.int32)
        w = rng.random((cap, k)).astype(np.float32)
        x[:n], ids[:n], w[:n] = d["x"][p:p + n], d["topk_ids"][p:p + n], d["topk_weights"][p:p + n]
        r = dict(d)
        r.update(T=cap, x=x, topk_ids=ids, topk_weights=w, n=n)
        reqs.append(r)
        p += n
    return d, reqs


def payload(r):
    """A request's payload arrays on the device (its whole buffer)."""
    x = torch.from_numpy(np.ascontiguousarray(r["x"]).view(np.int16)).view(torch.bfloat16).cuda()
    return (x, torch.from_numpy(np.ascontiguousarray(r["topk_ids"])).cuda(),
            torch.from_numpy(np.ascontiguousarray(r["topk_weights"])).cuda())


def _wdt(d, act8):
    if d["wdtype"] != "fp8":
        return eaas.EAAS_BF16
    return eaas.EAAS_FP8_E4M3_A8 if act8 else eaas.EAAS_FP8_E4M3


def run_segments(d, reqs, capacity, out_dtype=torch.float32, in_place=False, act8=False):
    """Device buffers for every request, then one segments call."""
    dev = to_device(d)
    bufs = []
    for r in reqs:
        x, ids, w = payload(r)
        if in_place:
            out = x
        else:
            out = torch.full((r["T"], d["H"]), float("nan"), dtype=out_dtype, device="cuda")
        bufs.append((x, ids, w, out))
    table = eaas.segment_table(bufs)
    counts = torch.tensor([r["n"] for r in reqs], dtype=torch.int32, device="cuda")
    ws = eaas.alloc_segments_workspace(capacity, d["H"], d["I"], d["E"], d["k"], _wdt(d, act8))
    odt = eaas.EAAS_FP32 if (out_dtype == torch.float32 and not in_place) else eaas.EAAS_BF16
    eaas.eaas_expert_forward_segments(table, counts, len(reqs), capacity, d["k"], dev["w_gate_up"],
                                      dev["w_down"], ws, odt, dev["w_gate_up_scale"],
                                      dev["w_down_scale"], act8=act8)
    torch.cuda.synchronize()
    return bufs, dict(table=table, counts=counts, ws=ws, dev=dev, odt=odt)


def forward_concat(d, reqs, out_dtype=torch.float32, limit=None, act8=False):
    """eaas_expert_forward on the requests concatenated in slot order."""
    cat = S.dynamic_batch(reqs)
    if limit is not None:
        cat = O.sub_batch(cat, range(min(limit, cat["T"])))
    if cat["T"] == 0:
        return np.zeros((0, d["H"]))
    dev = to_device(cat)
    ws = eaas.alloc_workspace(cat["T"], d["H"], d["I"], d["E"], d["k"], _wdt(d, act8))
    out = torch.empty((cat["T"], d["H"]), dtype=out_dtype, device="cuda")
    eaas.eaas_expert_forward(dev["x"], dev["topk_ids"], dev["topk_weights"], dev["w_gate_up"],
                             dev["w_down"], out, ws, dev["w_gate_up_scale"], dev["w_down_scale"],
                             act8=act8)
    torch.cuda.synchronize()
    return out


def check_against(reqs, bufs, ref, limit=None):
    """Rows [0, n) of each request equal the concatenated result bitwise;
    everything else of the out buffer is untouched (still NaN)."""
    p = 0
    for r, (_, _, _, out) in zip(reqs, bufs):
        n = r["n"]
        done = max(0, min(n, (limit if limit is not None else 1 << 30) - p))
        o = out.cpu()
        if done:
            assert torch.equal(o[:done].view(torch.int32), ref[p:p + done].cpu().view(torch.int32))
        assert torch.isnan(o[done:]).all(), "rows past the request were written"
        p += n


def check_oracle(reqs, bufs):
    ref = S.segmented_forward(reqs)
    for r, (_, _, _, out), g in zip(reqs, bufs, ref):
        if r["n"] == 0:
            continue
        got = out[: r["n"]].cpu().numpy().astype(np.float64)
        rms = float(np.sqrt((g ** 2).mean()))
        err = float(np.abs(got - g).max())
        assert err <= TOL * rms, (err, rms)


@pytest.mark.parametrize("sizes,capacity", [
    ([37, 0, 100, 1, 162], 320), ([5], 5), ([0, 0, 9], 64), ([64, 64, 64, 64], 256),
])
def test_segments_match_concatenated_forward(gpu, sizes, capacity):
    d, reqs = make_requests(sizes)
    say("segments bf16", sizes, capacity)
    bufs, _ = run_segments(d, reqs, capacity)
    check_against(reqs, bufs, forward_concat(d, reqs))
    check_oracle(reqs, bufs)


def test_segments_fp8_many_clients(gpu):
    rng = np.random.default_rng(9)
    sizes = [int(v) for v in rng.integers(0, 13, size=24)]
    d, reqs = make_requests(sizes, H=1024, I=512, E=16, k=8, seed=42, wdtype="fp8")
    say("segments fp8", sum(sizes))
    bufs, _ = run_segments(d, reqs, 256)
    check_against(reqs, bufs, forward_concat(d, reqs))
    check_oracle(reqs, bufs)


def test_segments_fp8_activations(gpu):
    # fp8 activations: x and h are quantized per row, so each request's rows
    # still equal the concatenated step's bit for bit
    rng = np.random.default_rng(11)
    sizes = [int(v) for v in rng.integers(0, 40, size=12)]
    d, reqs = make_requests(sizes, H=512, I=256, E=16, k=4, seed=44, wdtype="fp8")
    say("segments fp8 activations", sum(sizes))
    bufs, _ = run_segments(d, reqs, 512, act8=True)
    check_against(reqs, bufs, forward_concat(d, reqs, act8=True))


def test_fp8_activation_tile_heights_agree(gpu):
    """The fp8 x fp8 GEMMs take 128-row tiles when T*k <= 128*E and 192-row
    tiles above.  Here the concatenated batch (about 240 tokens, T*k <= 2048)
    takes the short tiles and the segmented step sized for 1024 tokens the
    tall ones; the per-block arithmetic is the same, so the bits agree."""
    rng = np.random.default_rng(12)
    sizes = [int(v) for v in rng.integers(0, 40, size=12)]
    d, reqs = make_requests(sizes, H=512, I=256, E=16, k=4, seed=45, wdtype="fp8")
    assert sum(sizes) * 4 <= 128 * 16 < 1024 * 4
    say("fp8 activations, 128- and 192-row tiles", sum(sizes))
    bufs, _ = run_segments(d, reqs, 1024, act8=True)
    check_against(reqs, bufs, forward_concat(d, reqs, act8=True))


def test_segments_capacity_cuts_the_batch(gpu):
    d, reqs = make_requests([50, 80, 40])
    say("segments capacity 100 of 170")
    bufs, _ = run_segments(d, reqs, 100)
    check_against(reqs, bufs, forward_concat(d, reqs, limit=100), limit=100)


def test_segments_negative_counts_are_empty(gpu):
    d, reqs = make_requests([10, 0, 12])
    say("segments negative count")
    dev = to_device(d)
    bufs = [payload(r) + (torch.full((r["T"], d["H"]), float("nan"), device="cuda"),)
            for r in reqs]
    table = eaas.segment_table(bufs)
    counts = torch.tensor([10, -4, 12], dtype=torch.int32, device="cuda")
    ws = eaas.alloc_segments_workspace(64, d["H"], d["I"], d["E"], d["k"])
    eaas.eaas_expert_forward_segments(table, counts, 3, 64, d["k"], dev["w_gate_up"], dev["w_down"],
                                      ws, eaas.EAAS_FP32)
    torch.cuda.synchronize()
    reqs[1]["n"] = 0
    check_against(reqs, bufs, forward_concat(d, reqs))


def test_segments_in_place_write_back(gpu):
    d, reqs = make_requests([20, 33, 0, 7])
    say("segments in place")
    bufs, _ = run_segments(d, reqs, 64, out_dtype=torch.bfloat16)
    ip, _ = run_segments(d, reqs, 64, in_place=True)
    for r, (_, _, _, out), (x, _, _, _) in zip(reqs, bufs, ip):
        n = r["n"]
        assert np.array_equal(bf16_tensor_to_bits(x[:n]), bf16_tensor_to_bits(out[:n]))
        # the payload rows past the request keep their hidden states
        assert np.array_equal(bf16_tensor_to_bits(x[n:]), r["x"][n:])


def test_segments_max_requests(gpu):
    rng = np.random.default_rng(10)
    sizes = [int(v) for v in rng.integers(0, 3, size=1024)]
    d, reqs = make_requests(sizes, H=256, I=128, E=8, k=2, seed=43, pad=1)
    say("segments 1024 requests", sum(sizes))
    bufs, _ = run_segments(d, reqs, 2048)
    check_against(reqs, bufs, forward_concat(d, reqs))


def test_segments_graph_replay_with_new_counts(gpu):
    d, reqs = make_requests([30, 20, 25, 10])
    say("segments graph replay")
    bufs, st = run_segments(d, reqs, 128)
    dev, table, counts, ws = st["dev"], st["table"], st["counts"], st["ws"]

    def call():
        eaas.eaas_expert_forward_segments(table, counts, len(reqs), 128, d["k"], dev["w_gate_up"],
                                          dev["w_down"], ws, eaas.EAAS_FP32)

    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        call()
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        call()
    for new in ([30, 20, 25, 10], [0, 20, 3, 10], [12, 0, 0, 1], [30, 20, 25, 10]):
        for r, n in zip(reqs, new):
            r["n"] = n
        counts.copy_(torch.tensor(new, dtype=torch.int32))
        for b in bufs:
            b[3].fill_(float("nan"))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        check_against(reqs, bufs, forward_concat(d, reqs))
