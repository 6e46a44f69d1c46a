"""C ABI host side, no GPU: the library loads, exports every declared symbol,
and rejects bad arguments on the host before touching the device."""
import ctypes
import os
import re

import pytest

from paper_2509_17863_amd import eaas

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    src = open(os.path.join(ROOT, "include", "eaas.h")).read()
    return sorted(set(re.findall(r"\b(eaas_[a-z0-9_]+)\s*\(", src)))


def test_header_declares_the_exported_set():
    assert _declared() == sorted(eaas.EXPORTED)


def test_library_exports_every_declared_symbol():
    L = eaas.lib()
    for name in _declared():
        assert hasattr(L, name), name


def test_status_strings():
    assert eaas.eaas_status_string(0) == "ok"
    assert "workspace" in eaas.eaas_status_string(-3)


def shape(T=64, H=256, I=128, E=8, k=2):
    return eaas._Shape(T, H, I, E, k)


@pytest.mark.parametrize("kw,ok", [
    (dict(), True), (dict(T=0), True), (dict(H=200), False), (dict(I=100), False),
    (dict(E=0), False), (dict(E=1025), False), (dict(k=0), False), (dict(k=65), False),
    (dict(T=-1), False), (dict(T=1 << 28, k=8), False),
    # 32-bit element offsets in the kernels: T*H, T*k*I and 4*I*H stay <= INT_MAX
    (dict(T=(1 << 24) - 1, H=128, I=128, k=1), True), (dict(T=1 << 24, H=128, I=128, k=1), False),
    (dict(T=(1 << 23) - 1, H=128, I=256, k=1), True), (dict(T=1 << 23, H=128, I=256, k=1), False),
    (dict(T=4, H=23168, I=23168), True), (dict(T=4, H=23168, I=23296), False),
])
def test_workspace_bytes_validation(kw, ok):
    s = shape(**kw)
    n = eaas.lib().eaas_workspace_bytes(ctypes.byref(s), 0)
    assert (n > 0) == ok
    if ok:
        assert n % 256 == 0
        assert eaas.lib().eaas_workspace_bytes(ctypes.byref(s), 7) == 0


def test_workspace_covers_stage_and_h():
    T, H, I, E, k = 100, 512, 256, 8, 4
    n = eaas.eaas_workspace_bytes(T, H, I, E, k)
    assert n >= T * k * H * 4 + T * k * I * 2


FAKE = 1 << 20  # host-only: these calls must be rejected before any device work


def _routing(p=FAKE):
    return eaas._Routing(p, p, p, p, p)


def test_route_permute_rejects_bad_args():
    L = eaas.lib()
    s = shape()
    r = _routing()
    assert L.eaas_route_permute(None, FAKE, ctypes.byref(r), FAKE, 1 << 30, None) == -1
    assert L.eaas_route_permute(ctypes.byref(s), None, ctypes.byref(r), FAKE, 1 << 30, None) == -1
    assert L.eaas_route_permute(ctypes.byref(s), FAKE, None, FAKE, 1 << 30, None) == -1
    assert L.eaas_route_permute(ctypes.byref(s), FAKE, ctypes.byref(r), None, 1 << 30, None) == -3
    assert L.eaas_route_permute(ctypes.byref(s), FAKE, ctypes.byref(r), FAKE, 16, None) == -3
    bad = shape(H=96)
    assert L.eaas_route_permute(ctypes.byref(bad), FAKE, ctypes.byref(r), FAKE, 1 << 30, None) == -2
    empty = shape(T=0)
    assert L.eaas_route_permute(ctypes.byref(empty), None, None, None, 0, None) == 0


def test_forward_rejects_bad_args():
    L = eaas.lib()
    s = shape()
    big = 1 << 34

    def fwd(x=FAKE, ids=FAKE, w=FAKE, wgu=FAKE, sgu=None, wd=FAKE, sd=None, wdt=0, out=FAKE * 64,
            odt=0, r=None, ws=FAKE, wsb=big, sh=s):
        return L.eaas_expert_forward(ctypes.byref(sh) if sh is not None else None, x, ids, w,
                                     wgu, sgu, wd, sd, wdt, out, odt, r, ws, wsb, None)

    assert fwd(sh=None) == -1
    assert fwd(x=None) == -1
    assert fwd(ids=None) == -1
    assert fwd(wgu=None) == -1
    assert fwd(wdt=1) == -1            # fp8 without scales
    assert fwd(wdt=5) == -1            # unknown weight dtype
    assert fwd(odt=1) == -1            # fp8 output is not offered
    assert fwd(x=FAKE + 8) == -1       # misaligned
    assert fwd(out=FAKE + 256) == -1   # partial overlap with x
    assert fwd(out=FAKE, odt=2) == -1  # fp32 output cannot alias bf16 x
    assert fwd(ws=None) == -3
    assert fwd(wsb=1024) == -3
    assert fwd(sh=shape(E=2000)) == -2
    assert fwd(sh=shape(T=0), x=None, ids=None) == 0


def test_ffn_and_combine_reject_bad_args():
    L = eaas.lib()
    s = shape()
    r = _routing()
    assert L.eaas_expert_ffn_grouped(ctypes.byref(s), FAKE, ctypes.byref(r), FAKE, None, FAKE,
                                     None, 1, FAKE, FAKE, 1 << 34, None) == -1
    assert L.eaas_expert_ffn_grouped(ctypes.byref(s), FAKE, ctypes.byref(r), FAKE, None, FAKE,
                                     None, 0, None, FAKE, 1 << 34, None) == -1
    assert L.eaas_unpermute_combine(ctypes.byref(s), FAKE, ctypes.byref(r), FAKE, FAKE, 1,
                                    None) == -1
    assert L.eaas_unpermute_combine(ctypes.byref(s), FAKE, ctypes.byref(r), None, FAKE, 0,
                                    None) == -1


def test_missing_library_fails_loudly(monkeypatch, tmp_path):
    monkeypatch.setattr(eaas, "_LIB_PATH", tmp_path / "libeaas.so")
    monkeypatch.setattr(eaas, "_lib", None)
    with pytest.raises(RuntimeError, match="missing"):
        eaas.lib()


def test_segments_workspace_exceeds_single_batch():
    T, H, I, E, k = 100, 512, 256, 8, 4
    single = eaas.eaas_workspace_bytes(T, H, I, E, k)
    seg = eaas.eaas_segments_workspace_bytes(T, H, I, E, k)
    # the gathered batch (x rows, ids, scores) comes on top
    assert seg >= single + T * H * 2 + 2 * T * k * 4
    s = shape(H=200)
    assert eaas.lib().eaas_segments_workspace_bytes(ctypes.byref(s), 0) == 0


def test_forward_segments_rejects_bad_args():
    L = eaas.lib()
    s = shape()
    ws = 1 << 30
    args = lambda **kw: dict(dict(s=ctypes.byref(s), segs=FAKE, n=FAKE, n_seg=3, wgu=FAKE, sgu=None,  # noqa: E731
                                  wd=FAKE, sd=None, wdt=0, odt=0, ws=FAKE, wsb=ws), **kw)

    def call(a):
        return L.eaas_expert_forward_segments(a["s"], a["segs"], a["n"], a["n_seg"], a["wgu"],
                                              a["sgu"], a["wd"], a["sd"], a["wdt"], a["odt"],
                                              a["ws"], a["wsb"], None)
    assert call(args(s=None)) == -1
    assert call(args(n_seg=-1)) == -1
    assert call(args(n_seg=1025)) == -1
    assert call(args(segs=None)) == -1
    assert call(args(n=None)) == -1
    assert call(args(odt=1)) == -1            # fp8 is not an output type
    assert call(args(wdt=1)) == -1            # fp8 weights without scales
    assert call(args(wgu=FAKE + 8)) == -1     # misaligned weights
    assert call(args(ws=None)) == -3
    assert call(args(wsb=64)) == -3
    bad = shape(I=100)
    assert call(args(s=ctypes.byref(bad))) == -2
    # nothing to do: no requests, or no capacity
    assert call(args(n_seg=0, segs=None, n=None)) == 0
    empty = shape(T=0)
    assert call(args(s=ctypes.byref(empty), segs=None, n=None)) == 0


def test_server_workspace_and_validation():
    L = eaas.lib()
    s = shape(E=32)
    assert L.eaas_server_workspace_bytes(ctypes.byref(s), 32, 0) > 0
    assert L.eaas_server_workspace_bytes(ctypes.byref(s), 33, 0) == 0   # 33*32 groups > 1024
    assert L.eaas_server_workspace_bytes(ctypes.byref(s), 0, 0) == 0
    assert L.eaas_server_workspace_bytes(ctypes.byref(s), 2, 2) == 0    # fp32 weights
    ws = 1 << 30

    def call(s_=ctypes.byref(s), slots=FAKE, n=4, layers=FAKE, nl=2, wdt=0, w=FAKE, wb=ws):
        return L.eaas_server_step(s_, slots, n, layers, nl, wdt, w, wb, None)
    assert call(s_=None) == -1
    assert call(n=-1) == -1
    assert call(n=1025) == -1
    assert call(slots=None) == -1
    assert call(layers=None) == -1
    assert call(nl=0) == -1
    assert call(nl=40) == -2
    assert call(wdt=2) == -1
    assert call(w=None) == -3
    assert call(wb=128) == -3
    assert call(n=0, slots=None, layers=None) == 0


def test_fp8_activation_mode_host_validation():
    L = eaas.lib()
    A8 = eaas.EAAS_FP8_E4M3_A8
    # H must be a multiple of 256 (the down projection's 256-wide N tiles)
    assert eaas.eaas_workspace_bytes(64, 384, 128, 8, 2, A8) == 0
    n8 = eaas.eaas_workspace_bytes(64, 512, 128, 8, 2, eaas.EAAS_FP8_E4M3)
    na8 = eaas.eaas_workspace_bytes(64, 512, 128, 8, 2, A8)
    assert na8 >= n8 + 64 * 512 + 64 * 4 * 4  # + quantized x and its scales
    s = shape(H=512)
    big = 1 << 34

    def fwd(wdt=A8, sgu=FAKE, sd=FAKE, sh=s):
        return L.eaas_expert_forward(ctypes.byref(sh), FAKE, FAKE, FAKE, FAKE, sgu, FAKE, sd, wdt,
                                     FAKE * 64, 0, None, FAKE, big, None)

    assert fwd(sgu=None) == -1            # fp8 weights need their scales
    assert fwd(sh=shape(H=384)) == -2     # H not a multiple of 256
    # the batched entry points take fp8 activations with the same limits
    assert L.eaas_segments_workspace_bytes(ctypes.byref(s), A8) > na8
    assert L.eaas_server_workspace_bytes(ctypes.byref(s), 2, A8) > 0
    bad = shape(H=384)
    assert L.eaas_segments_workspace_bytes(ctypes.byref(bad), A8) == 0
    assert L.eaas_server_workspace_bytes(ctypes.byref(bad), 1, A8) == 0
    assert L.eaas_expert_forward_segments(ctypes.byref(bad), FAKE, FAKE, 1, FAKE, FAKE, FAKE,
                                          FAKE, A8, 0, FAKE, big, None) == -2
    assert L.eaas_server_step(ctypes.byref(bad), FAKE, 1, FAKE, 1, A8, FAKE, big, None) == -2


def test_quantize_rows_rejects_bad_args():
    L = eaas.lib()
    assert L.eaas_quantize_rows_fp8(FAKE, -1, 128, FAKE, FAKE, None) == -1
    assert L.eaas_quantize_rows_fp8(FAKE, 4, 0, FAKE, FAKE, None) == -1
    assert L.eaas_quantize_rows_fp8(FAKE, 4, 100, FAKE, FAKE, None) == -2
    assert L.eaas_quantize_rows_fp8(FAKE, 1 << 24, 1 << 10, FAKE, FAKE, None) == -2
    assert L.eaas_quantize_rows_fp8(None, 4, 128, FAKE, FAKE, None) == -1
    assert L.eaas_quantize_rows_fp8(FAKE + 8, 4, 128, FAKE, FAKE, None) == -1
    assert L.eaas_quantize_rows_fp8(FAKE, 4, 128, None, FAKE, None) == -1
    assert L.eaas_quantize_rows_fp8(None, 0, 128, None, None, None) == 0


@pytest.mark.parametrize("T,H,I,E,k,wdt", [(64, 256, 128, 8, 2, 0), (16384, 7168, 2048, 32, 8, 0),
                                          (256, 7168, 2048, 32, 8, 1), (300, 512, 256, 6, 2, 3),
                                          (5000, 2048, 768, 128, 8, 0)])
def test_workspace_bytes_per_entry(T, H, I, E, k, wdt):
    """route_permute needs its histogram, ffn_grouped everything but the
    staging, the forward the whole workspace."""
    f = lambda e: eaas.eaas_workspace_bytes_for(T, H, I, E, k, wdt, e)  # noqa: E731
    route, ffn, fwd = (f(eaas.EAAS_ENTRY_ROUTE_PERMUTE), f(eaas.EAAS_ENTRY_FFN_GROUPED),
                       f(eaas.EAAS_ENTRY_FORWARD))
    R = T * k
    assert fwd == eaas.eaas_workspace_bytes(T, H, I, E, k, wdt)
    assert route == -(-((R + 2047) // 2048) * E * 4 // 256) * 256
    assert route < ffn < fwd
    assert ffn >= R * I * 2 + 2 * R * 4
    assert fwd - ffn >= R * H * 4                 # the fp32 staging is the forward's alone
    assert eaas.eaas_workspace_bytes_for(T, H, I, E, k, wdt, 7) == 0
    assert eaas.eaas_workspace_bytes_for(T, 200, I, E, k, wdt, 0) == 0


def test_entry_workspace_minimums_enforced():
    L = eaas.lib()
    s = shape()
    r = _routing()
    route = eaas.eaas_workspace_bytes_for(64, 256, 128, 8, 2, 0, eaas.EAAS_ENTRY_ROUTE_PERMUTE)
    ffn = eaas.eaas_workspace_bytes_for(64, 256, 128, 8, 2, 0, eaas.EAAS_ENTRY_FFN_GROUPED)
    assert L.eaas_route_permute(ctypes.byref(s), FAKE, ctypes.byref(r), FAKE, route - 1,
                                None) == -3
    assert L.eaas_route_permute(ctypes.byref(s), FAKE, ctypes.byref(r), FAKE + 8, route,
                                None) == -3   # misaligned workspace
    assert L.eaas_expert_ffn_grouped(ctypes.byref(s), FAKE, ctypes.byref(r), FAKE, None, FAKE,
                                     None, 0, FAKE, FAKE, ffn - 1, None) == -3


def test_k_above_E_is_a_valid_shape():
    """A server may hold fewer experts than a token has slots (the other
    slots name experts of other servers and are skipped): k > E passes
    validation, up to the k <= 64 limit."""
    assert eaas.eaas_workspace_bytes(64, 256, 128, 3, 8) > 0
    assert eaas.eaas_workspace_bytes(64, 256, 128, 1, 64) > 0
    assert eaas.eaas_workspace_bytes(64, 256, 128, 1, 65) == 0
    L = eaas.lib()
    s = shape(E=3, k=8)
    r = _routing()
    # validation passes the shape and stops at the missing workspace
    assert L.eaas_route_permute(ctypes.byref(s), FAKE, ctypes.byref(r), None, 0, None) == -3


def test_tiled_fp8_dtype_and_tile_entry_validation():
    """EAAS_FP8_E4M3_TILED: the fp8 workspace, H a multiple of 256; the
    tiling entry point rejects bad arguments on the host."""
    T8 = eaas.EAAS_FP8_E4M3_TILED
    assert eaas.eaas_workspace_bytes(64, 512, 256, 8, 2, T8) == \
        eaas.eaas_workspace_bytes(64, 512, 256, 8, 2, eaas.EAAS_FP8_E4M3)
    assert eaas.eaas_workspace_bytes(64, 384, 256, 8, 2, T8) == 0
    L = eaas.lib()
    s = shape(H=512, I=256)
    assert L.eaas_tile_weights_fp8(None, 0, FAKE, FAKE * 64, None) == -1
    assert L.eaas_tile_weights_fp8(ctypes.byref(s), 2, FAKE, FAKE * 64, None) == -1
    assert L.eaas_tile_weights_fp8(ctypes.byref(s), 0, None, FAKE * 64, None) == -1
    assert L.eaas_tile_weights_fp8(ctypes.byref(s), 0, FAKE + 8, FAKE * 64, None) == -1
    assert L.eaas_tile_weights_fp8(ctypes.byref(s), 0, FAKE, FAKE + 4096, None) == -1  # overlap
    assert L.eaas_tile_weights_fp8(ctypes.byref(s), 1, FAKE, FAKE, None) == -1         # in place
    bad = shape(H=384, I=256)
    assert L.eaas_tile_weights_fp8(ctypes.byref(bad), 0, FAKE, FAKE * 64, None) == -2
    # the fp8 scales are required as for row-major fp8 weights
    big = 1 << 34
    assert L.eaas_expert_forward(ctypes.byref(s), FAKE, FAKE, FAKE, FAKE, None, FAKE, None, T8,
                                 FAKE * 64, 0, None, FAKE, big, None) == -1
