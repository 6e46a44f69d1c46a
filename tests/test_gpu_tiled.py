"""fp8 weights in the tiled layout (EAAS_FP8_E4M3_TILED) through the C ABI:
the layout eaas_tile_weights_fp8 writes matches its definition (a plain NumPy
rearrangement written from the header), and every entry point gives the same
results, bit for bit, as with the row-major weights.  Every case prints its
name before touching the GPU."""
import numpy as np
import pytest
import torch

from paper_2509_17863_amd import eaas, synth
from paper_2509_17863_amd.device_io import to_device

pytestmark = pytest.mark.gpu


def say(*a):
    print("[gpu-case]", *a, flush=True)


def tiled_reference(w, which, I):
    """The tiled layout from its definition: per expert, N tile and 64-byte
    K tile, the tile's rows (gate rows before up rows) one after the other."""
    E, N, K = w.shape
    BN = 512 if which == eaas.EAAS_GATE_UP and N % 512 == 0 else 256
    out = np.empty(E * N * K, np.uint8)
    pos = 0
    for e in range(E):
        for tn in range(N // BN):
            if which == eaas.EAAS_GATE_UP:
                rows = np.concatenate([tn * BN // 2 + np.arange(BN // 2),
                                       I + tn * BN // 2 + np.arange(BN // 2)])
            else:
                rows = tn * BN + np.arange(BN)
            for kt in range(K // 64):
                blk = w[e, rows, kt * 64:(kt + 1) * 64]
                out[pos:pos + blk.size] = blk.reshape(-1)
                pos += blk.size
    return out.reshape(E, N, K)


def tile(dev_w, which, H, I):
    out = torch.empty_like(dev_w)
    eaas.eaas_tile_weights_fp8(dev_w, which, H, I, out)
    return out


@pytest.mark.parametrize("E,H,I", [(3, 512, 256), (2, 768, 384), (2, 256, 512)])
def test_tile_layout_matches_definition(gpu, E, H, I):
    rng = np.random.default_rng(E * H + I)
    wgu = rng.integers(0, 256, size=(E, 2 * I, H), dtype=np.uint8)
    wdn = rng.integers(0, 256, size=(E, H, I), dtype=np.uint8)
    say("tile layout", E, H, I)
    for which, w in ((eaas.EAAS_GATE_UP, wgu), (eaas.EAAS_DOWN, wdn)):
        got = tile(torch.from_numpy(w).cuda(), which, H, I).cpu().numpy()
        assert np.array_equal(got, tiled_reference(w, which, I)), which


def tiled_dev(d):
    dev = to_device(d)
    H, I = d["H"], d["I"]
    dev = dict(dev)
    dev["w_gate_up"] = tile(dev["w_gate_up"], eaas.EAAS_GATE_UP, H, I)
    dev["w_down"] = tile(dev["w_down"], eaas.EAAS_DOWN, H, I)
    return dev


def forward(dev, k, tiled, out_dtype=torch.float32, noalloc=False):
    T, H = dev["x"].shape
    E, twoI, _ = dev["w_gate_up"].shape
    out = torch.full((T, H), float("nan"), dtype=out_dtype, device="cuda")
    if noalloc:
        eaas.eaas_expert_forward_noalloc(dev["x"], dev["topk_ids"], dev["topk_weights"],
                                         dev["w_gate_up"], dev["w_down"], out,
                                         dev["w_gate_up_scale"], dev["w_down_scale"], tiled=tiled)
        return out
    wdt = eaas.EAAS_FP8_E4M3_TILED if tiled else eaas.EAAS_FP8_E4M3
    ws = eaas.alloc_workspace(T, H, twoI // 2, E, k, wdt)
    eaas.eaas_expert_forward(dev["x"], dev["topk_ids"], dev["topk_weights"], dev["w_gate_up"],
                             dev["w_down"], out, ws, dev["w_gate_up_scale"], dev["w_down_scale"],
                             tiled=tiled)
    return out


CASES = [
    # T, H, I, E, k, seed, zipf, mask
    (256, 7168, 2048, 32, 8, 4, None, 0.0),    # the decode workload's shape: gate/up BN 512
    (300, 768, 384, 6, 3, 91, 1.3, 0.1),       # gate/up 2I = 768: BN 256; ragged, masked
    (900, 512, 256, 4, 2, 92, None, 0.0),      # several M tiles per expert
]


@pytest.mark.parametrize("T,H,I,E,k,seed,zipf,mask", CASES)
def test_tiled_forward_equals_row_major(gpu, T, H, I, E, k, seed, zipf, mask):
    d = synth.make_inputs(T, H, I, E, k, seed, zipf=zipf, wdtype="fp8")
    if mask:
        rng = np.random.default_rng(seed)
        ids = d["topk_ids"].copy()
        ids[rng.random(ids.shape) < mask] = -1
        d["topk_ids"] = ids
    say("tiled forward", T, H, I, E, k)
    dev = to_device(d)
    devt = tiled_dev(d)
    a = forward(dev, k, False)
    b = forward(devt, k, True)
    c = forward(devt, k, True, out_dtype=torch.bfloat16, noalloc=T * H <= 256 * 7168)
    ref16 = forward(dev, k, False, out_dtype=torch.bfloat16)
    torch.cuda.synchronize()
    assert torch.equal(a.view(torch.int32), b.view(torch.int32))
    assert torch.equal(c.view(torch.int16), ref16.view(torch.int16))


def test_tiled_modular_and_server_step(gpu):
    """The grouped FFN entry point and a server step over two layers of
    tiled weights, against the same calls with row-major weights."""
    from test_gpu_server import H as SH, I as SI, E as SE, K as SK, Server, make_layers, \
        make_slots, snapshot

    d = synth.make_inputs(200, 512, 256, 5, 3, 93, zipf=1.1, wdtype="fp8")
    T, H, I, E, k = d["T"], d["H"], d["I"], d["E"], d["k"]
    dev, devt = to_device(d), tiled_dev(d)
    say("tiled grouped FFN")
    ys = []
    for dv, tiled in ((dev, False), (devt, True)):
        wdt = eaas.EAAS_FP8_E4M3_TILED if tiled else eaas.EAAS_FP8_E4M3
        r = eaas.alloc_routing(T, k, E)
        ws = eaas.alloc_workspace(T, H, I, E, k, wdt)
        eaas.eaas_route_permute(dv["topk_ids"], E, r, ws, H=H, I=I)
        y = torch.zeros((T * k, H), dtype=torch.float32, device="cuda")
        eaas.eaas_expert_ffn_grouped(dv["x"], r, dv["w_gate_up"], dv["w_down"], y, ws, k,
                                     dv["w_gate_up_scale"], dv["w_down_scale"], tiled=tiled)
        ys.append(y)
    torch.cuda.synchronize()
    assert torch.equal(ys[0].view(torch.int32), ys[1].view(torch.int32))

    say("tiled server step")
    layers = make_layers(2, wdtype="fp8", seed=94)
    specs = [(1, L % 2, n, n + 2) for L, n in enumerate([19, 7, 33, 0, 12])]
    results = []
    for tiled in (False, True):
        srv = Server(make_slots(specs, seed=95), layers, capacity=128)
        if tiled:
            for dl in srv.dl:
                dl["w_gate_up"] = tile(dl["w_gate_up"], eaas.EAAS_GATE_UP, SH, SI)
                dl["w_down"] = tile(dl["w_down"], eaas.EAAS_DOWN, SH, SI)
            srv.ltab = eaas.layer_table([(x["w_gate_up"], x["w_gate_up_scale"], x["w_down"],
                                          x["w_down_scale"]) for x in srv.dl])
            srv.wdt = eaas.EAAS_FP8_E4M3_TILED
        srv.step()
        results.append(srv.state())
    assert results[0][0] == results[1][0]
    for a, b in zip(results[0][1], results[1][1]):
        assert np.array_equal(a, b)
