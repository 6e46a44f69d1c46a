"""The allocation-free forward (eaas_expert_forward_noalloc) through the C
ABI: the same results, bit for bit, as eaas_expert_forward with a workspace,
on two calls in a row (the second smaller, so it runs on what the first left
in the shared scratch array), and host-side rejection of shapes that need more
scratch than the library holds.  Every case prints its name before touching
the GPU."""
import ctypes

import numpy as np
import pytest
import torch

from paper_2509_17863_amd import eaas, synth
from paper_2509_17863_amd.device_io import to_device


def say(*a):
    print("[gpu-case]", *a, flush=True)


def with_workspace(dev, k, act8, out_dtype):
    T, H = dev["x"].shape
    E, twoI, _ = dev["w_gate_up"].shape
    wdt = eaas._wdtype(dev["w_gate_up"], act8)
    ws = eaas.alloc_workspace(T, H, twoI // 2, E, k, wdt)
    out = torch.full((T, H), float("nan"), dtype=out_dtype, device="cuda")
    eaas.eaas_expert_forward(dev["x"], dev["topk_ids"], dev["topk_weights"], dev["w_gate_up"],
                             dev["w_down"], out, ws, dev["w_gate_up_scale"], dev["w_down_scale"],
                             act8=act8)
    return out


def no_alloc(dev, act8, out_dtype, routing=None):
    T, H = dev["x"].shape
    out = torch.full((T, H), float("nan"), dtype=out_dtype, device="cuda")
    eaas.eaas_expert_forward_noalloc(dev["x"], dev["topk_ids"], dev["topk_weights"],
                                     dev["w_gate_up"], dev["w_down"], out, dev["w_gate_up_scale"],
                                     dev["w_down_scale"], routing=routing, act8=act8)
    return out


def bits(t):
    return t.cpu().contiguous().view(torch.int32 if t.dtype == torch.float32 else torch.int16).numpy()


@pytest.mark.gpu
@pytest.mark.parametrize("mode", ["fp8", "bf16", "fp8_act"])
def test_noalloc_matches_workspace_forward_twice(gpu, mode):
    wdtype = "bf16" if mode == "bf16" else "fp8"
    act8 = mode == "fp8_act"
    # first call: the decode-sized step (T 256, H 7168, I 2048, 32 experts, top 8)
    big = synth.make_inputs(256, 7168, 2048, 32, 8, 4, wdtype=wdtype)
    # second call, smaller: other experts, ragged tiles, masked slots
    small = synth.make_inputs(150, 512, 256, 6, 3, 5, zipf=1.2, wdtype=wdtype)
    small["topk_ids"][::7, 2] = -1
    for name, d, odt in (("decode-sized", big, torch.bfloat16), ("smaller", small, torch.float32)):
        dev = to_device(d)
        say("noalloc", mode, name)
        ref = with_workspace(dev, d["k"], act8, odt)
        r = eaas.alloc_routing(d["T"], d["k"], d["E"])
        got = no_alloc(dev, act8, odt, routing=r if name == "smaller" else None)
        torch.cuda.synchronize()
        assert np.array_equal(bits(got), bits(ref)), f"{mode} {name}: differs from the workspace call"
        if name == "smaller":
            from oracle import eaas_oracle as O
            ro = O.route_permute(d["topk_ids"], d["E"])
            R = d["T"] * d["k"]
            for key, n in (("counts", d["E"]), ("offsets", d["E"] + 1), ("perm", R), ("inv", R),
                           ("active", d["E"] + 1)):
                assert np.array_equal(r[key].cpu().numpy()[:n], ro[key]), key


@pytest.mark.gpu
def test_noalloc_in_place_and_graph_replay(gpu):
    """Written back into the payload (out == x), and captured in a graph:
    every replay, with eager work between replays, gives the eager result."""
    d = synth.make_inputs(96, 1024, 512, 8, 4, 6, wdtype="bf16")
    dev = to_device(d)
    say("noalloc in place + graph")
    ref = with_workspace(dev, d["k"], False, torch.bfloat16)
    x2 = dev["x"].clone()
    eaas.eaas_expert_forward_noalloc(x2, dev["topk_ids"], dev["topk_weights"], dev["w_gate_up"],
                                     dev["w_down"], x2)
    torch.cuda.synchronize()
    assert np.array_equal(bits(x2), bits(ref))
    out = torch.empty_like(ref)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        eaas.eaas_expert_forward_noalloc(dev["x"], dev["topk_ids"], dev["topk_weights"],
                                         dev["w_gate_up"], dev["w_down"], out)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        eaas.eaas_expert_forward_noalloc(dev["x"], dev["topk_ids"], dev["topk_weights"],
                                         dev["w_gate_up"], dev["w_down"], out)
    for i in range(3):
        out.fill_(float("nan"))
        with_workspace(dev, d["k"], False, torch.bfloat16)   # other work between replays
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert np.array_equal(bits(out), bits(ref)), i


def test_noalloc_rejects_shapes_beyond_its_scratch():
    """Host-side: a shape needing more than EAAS_NOALLOC_SCRATCH_BYTES is
    refused with EAAS_ERR_WORKSPACE before anything touches the device."""
    L = eaas.lib()
    fake = 1 << 20
    big = eaas._Shape(16384, 7168, 2048, 32, 8)
    assert eaas.eaas_workspace_bytes(16384, 7168, 2048, 32, 8) > eaas.EAAS_NOALLOC_SCRATCH_BYTES
    assert L.eaas_expert_forward_noalloc(ctypes.byref(big), fake, fake, fake, fake, None, fake,
                                         None, 0, fake * 64, 0, None, None) == -3
    bad = eaas._Shape(64, 200, 128, 8, 2)
    assert L.eaas_expert_forward_noalloc(ctypes.byref(bad), fake, fake, fake, fake, None, fake,
                                         None, 0, fake * 64, 0, None, None) == -2
    empty = eaas._Shape(0, 256, 128, 8, 2)
    assert L.eaas_expert_forward_noalloc(ctypes.byref(empty), None, None, None, None, None, None,
                                         None, 0, None, 0, None, None) == 0
    assert eaas.eaas_workspace_bytes(256, 7168, 2048, 32, 8, eaas.EAAS_FP8_E4M3_A8) <= \
        eaas.EAAS_NOALLOC_SCRATCH_BYTES
