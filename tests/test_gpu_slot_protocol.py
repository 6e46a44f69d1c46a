"""Host-driven tests of the slot protocol around the server step (EaaS §3.2
buffer states, §3.3 asynchronous server operation, §3.4 fault tolerance):

  * a late write: a client sets its slot ready on another stream while a step
    is in flight; the slot ends either answered whole (flag 2, every row the
    forward of the posted request) or untouched and still ready (flag 1, the
    payload exactly as posted), and the next step takes it;
  * a client's poll timeout: the server holding the request never steps, the
    client drops it from its expert-to-server mapping and re-sends the request
    to a replica, whose answer equals the forward of the request;
  * a monitor that stops hearing a client's heartbeat has the server release
    that client's slot (flag 3): the step leaves it alone and serves the rest;
    a client registering in the slot later is served again.

The host does all waiting, against bounded deadlines; no kernel spins.
Every case prints its name before touching the GPU.
"""
import time

import numpy as np
import pytest
import torch

from paper_2509_17863_amd import eaas
from paper_2509_17863_amd.device_io import bf16_tensor_to_bits
from test_gpu_server import (Server, check_step, forward_layer_concat, make_layers, make_slots,
                             say, snapshot)

pytestmark = pytest.mark.gpu


def stage_request(req):
    """A client's request held on the device, ready to be copied into a slot."""
    x = torch.from_numpy(req["x"].view(np.int16)).view(torch.bfloat16).cuda()
    return dict(x=x, ids=torch.from_numpy(req["topk_ids"]).cuda(),
                w=torch.from_numpy(req["topk_weights"]).cuda(),
                hdr=torch.tensor([req["layer"], req["n"]], dtype=torch.int32, device="cuda"))


def post_async(srv, b, st):
    """The client's write into slot b on the current stream: payload and
    header first, then the ready flag (stream order makes the payload visible
    before the flag)."""
    _, hdr, x, ids, w = srv.dev[b]
    n = st["x"].shape[0]
    x[:n].copy_(st["x"])
    ids[:n].copy_(st["ids"])
    w[:n].copy_(st["w"])
    hdr.copy_(st["hdr"])
    srv.dev[b][0].fill_(eaas.EAAS_SLOT_READY)


@pytest.mark.parametrize("client_first", [False, True])
@pytest.mark.parametrize("delay", [0, 2, 5, 13])
def test_late_write_is_answered_whole_or_left_ready(gpu, delay, client_first):
    """Which of the two outcomes occurs depends on when the runtime runs the
    two streams' work (they may share a hardware queue, which then runs them
    in submission order): the client's post is submitted after the step, or
    (client_first) before it, each behind `delay` matrix products."""
    layers = make_layers(1, seed=90)
    # slot 2 starts empty; its client posts while the step may be running
    specs = [(1, 0, 100, 128), (1, 0, 90, 96), (0, 0, 0, 64), (1, 0, 60, 64)]
    srv = Server(make_slots(specs, seed=91 + delay), layers, capacity=512)
    late = make_slots([(1, 0, 50, 64)], seed=200 + delay)[0]
    late["x"] = late["x"][:50]
    late["topk_ids"] = late["topk_ids"][:50]
    late["topk_weights"] = late["topk_weights"][:50]
    st = stage_request(late)
    big = torch.randn(2048, 2048, device="cuda")
    before = snapshot(srv.slots)
    torch.cuda.synchronize()
    say("late write, delay", delay, "client first" if client_first else "server first")
    sa, sb = torch.cuda.Stream(), torch.cuda.Stream()

    def server():
        with torch.cuda.stream(sa):
            for _ in range(4):
                big @ big
            srv.step(sa)

    def client():
        with torch.cuda.stream(sb):
            for _ in range(delay):
                big @ big
            post_async(srv, 2, st)

    for f in ((client, server) if client_first else (server, client)):
        f()
    torch.cuda.synchronize()
    flag = int(srv.dev[2][0].item())
    assert flag in (eaas.EAAS_SLOT_READY, eaas.EAAS_SLOT_DONE), flag
    x2 = bf16_tensor_to_bits(srv.dev[2][2])
    posted = dict(before[2], flag=eaas.EAAS_SLOT_READY, layer=0, n=50,
                  x=np.concatenate([late["x"], before[2]["x"][50:]]),
                  topk_ids=np.concatenate([late["topk_ids"], before[2]["topk_ids"][50:]]),
                  topk_weights=np.concatenate([late["topk_weights"],
                                               before[2]["topk_weights"][50:]]))
    srv.slots[2].update(layer=0, n=50, topk_ids=posted["topk_ids"],
                        topk_weights=posted["topk_weights"])
    if flag == eaas.EAAS_SLOT_DONE:
        say("late write, delay", delay, ": taken by the step in flight")
        check_step(srv, before[:2] + [posted] + before[3:])
        return
    say("late write, delay", delay, ": left ready for the next step")
    # untouched: the payload is exactly what the client wrote
    assert np.array_equal(x2, posted["x"])
    # the other slots as if slot 2 had stayed empty (its flag is the client's)
    srv.dev[2][0].fill_(eaas.EAAS_SLOT_EMPTY)
    check_step(srv, before[:2] + [dict(before[2], x=posted["x"])] + before[3:])
    srv.dev[2][0].fill_(eaas.EAAS_SLOT_READY)
    srv.slots[2]["flag"] = eaas.EAAS_SLOT_READY
    before2 = snapshot(srv.slots)
    srv.step()
    check_step(srv, before2)
    assert srv.slots[2]["flag"] == eaas.EAAS_SLOT_DONE


class Client:
    """An attention client's side of the protocol: it posts a request into
    its slot on the first server of its expert-to-server mapping, polls the
    slot's flag until a deadline, and on a timeout removes that server from
    the mapping and re-sends the request to the next replica (§3.4)."""

    def __init__(self, mapping, slot_of, pump, timeout_s):
        self.mapping, self.slot_of, self.pump, self.timeout_s = mapping, slot_of, pump, timeout_s
        self.dropped = []

    def submit(self, layer, req):
        st = stage_request(req)
        while self.mapping[layer]:
            srv = self.mapping[layer][0]
            b = self.slot_of[id(srv)]
            post_async(srv, b, st)
            torch.cuda.synchronize()
            deadline = time.monotonic() + self.timeout_s
            while time.monotonic() < deadline:
                self.pump()
                if int(srv.dev[b][0].item()) == eaas.EAAS_SLOT_DONE:
                    n = req["n"]
                    out = bf16_tensor_to_bits(srv.dev[b][2])[:n]
                    srv.dev[b][0].fill_(eaas.EAAS_SLOT_EMPTY)   # results read
                    return srv, out
                time.sleep(0.002)
            self.dropped.append(srv)
            self.mapping[layer].pop(0)
        raise TimeoutError("no live server holds the layer")


def test_client_timeout_fails_over_to_replica(gpu):
    layers = make_layers(1, seed=95)
    a = Server(make_slots([(0, 0, 0, 48)], seed=97), layers, capacity=64)
    b = Server(make_slots([(0, 0, 0, 48)], seed=98), layers, capacity=64)
    alive = {id(a): False, id(b): True}          # server a has died

    def pump():                                 # the live servers' loops
        for srv in (a, b):
            if alive[id(srv)]:
                srv.step()

    req = make_slots([(1, 0, 40, 48)], seed=96)[0]
    req["x"], req["topk_ids"], req["topk_weights"] = (req["x"][:40], req["topk_ids"][:40],
                                                      req["topk_weights"][:40])
    client = Client({0: [a, b]}, {id(a): 0, id(b): 0}, pump, timeout_s=0.25)
    say("client timeout and failover")
    t0 = time.monotonic()
    srv, out = client.submit(0, req)
    waited = time.monotonic() - t0
    assert srv is b and client.dropped == [a] and client.mapping[0] == [b]
    assert waited >= 0.25
    ref = forward_layer_concat([dict(req)], [0], [40], layers[0])
    assert np.array_equal(out, ref)
    # the dead server's slot holds the request untouched, still ready
    assert int(a.dev[0][0].item()) == eaas.EAAS_SLOT_READY
    assert np.array_equal(bf16_tensor_to_bits(a.dev[0][2])[:40], req["x"])
    # with no live replica left the client gives up after the deadline
    alive[id(b)] = False
    with pytest.raises(TimeoutError):
        client.submit(0, req)
    assert client.mapping[0] == []


class Monitor:
    """Heartbeat tracking (§3.4): a client silent for longer than `limit`
    is reported offline, and every server releases its slot (flag 3)."""

    def __init__(self, limit):
        self.limit, self.last, self.offline = limit, {}, set()

    def heartbeat(self, client, now):
        self.last[client] = now
        self.offline.discard(client)

    def sweep(self, now, servers):
        gone = [c for c, t in self.last.items() if now - t > self.limit and c not in self.offline]
        for c in gone:
            self.offline.add(c)
            for srv in servers:
                srv.dev[c][0].fill_(eaas.EAAS_SLOT_OFFLINE)
                srv.slots[c]["flag"] = eaas.EAAS_SLOT_OFFLINE
        return gone


def test_monitor_releases_the_slot_of_a_silent_client(gpu):
    layers = make_layers(1, seed=99)
    specs = [(1, 0, 30, 32), (1, 0, 25, 32), (1, 0, 20, 32), (1, 0, 10, 32)]
    srv = Server(make_slots(specs, seed=100), layers, capacity=128)
    mon = Monitor(limit=3.0)
    for c in range(4):
        mon.heartbeat(c, now=0.0)
    for now in (2.0, 4.0):                        # client 2 posted, then went silent
        for c in (0, 1, 3):
            mon.heartbeat(c, now)
    say("monitor releases a silent client's slot")
    assert mon.sweep(now=4.5, servers=[srv]) == [2]
    torch.cuda.synchronize()
    before = snapshot(srv.slots)
    srv.step()
    check_step(srv, before)
    assert [s["flag"] for s in srv.slots] == [2, 2, 3, 2]
    # a new client registers in the slot: the server resets it, the client posts
    mon.heartbeat(2, now=6.0)
    srv.dev[2][0].fill_(eaas.EAAS_SLOT_EMPTY)
    srv.slots[2]["flag"] = eaas.EAAS_SLOT_EMPTY
    srv.post(2, eaas.EAAS_SLOT_READY, 0, 20)
    torch.cuda.synchronize()
    before = snapshot(srv.slots)
    srv.step()
    check_step(srv, before)
    assert srv.slots[2]["flag"] == eaas.EAAS_SLOT_DONE
