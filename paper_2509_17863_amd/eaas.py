"""Python binding of libeaas.so: argument marshalling for the C ABI in
include/eaas.h, nothing else.  Every step of the forward pass runs in the HIP
kernels of the library; torch tensors are used only as device buffers and
torch streams as HIP streams.  There is no CPU fallback: if the library is not
built, every call raises.
"""
from __future__ import annotations

import ctypes
from pathlib import Path

import torch

__all__ = [
    "EAAS_OK", "EAAS_BF16", "EAAS_FP8_E4M3", "EAAS_FP32", "EAAS_FP8_E4M3_A8", "EaasError", "lib",
    "library_path", "eaas_workspace_bytes", "eaas_route_permute",
    "eaas_expert_ffn_grouped", "eaas_unpermute_combine", "eaas_expert_forward",
    "eaas_status_string", "eaas_expert_forward_profiled", "alloc_routing",
    "alloc_workspace", "EXPORTED", "eaas_segments_workspace_bytes",
    "alloc_segments_workspace", "segment_table", "eaas_expert_forward_segments",
    "EAAS_SLOT_EMPTY", "EAAS_SLOT_READY", "EAAS_SLOT_DONE", "EAAS_SLOT_OFFLINE",
    "eaas_server_workspace_bytes", "alloc_server_workspace", "slot_table", "layer_table",
    "eaas_server_step", "eaas_quantize_rows_fp8", "eaas_workspace_region", "workspace_view",
    "EAAS_WS_H", "EAAS_WS_HQ", "EAAS_WS_HS", "EAAS_WS_XQ", "EAAS_WS_XS", "EAAS_WS_STAGE",
    "eaas_workspace_bytes_for", "EAAS_ENTRY_ROUTE_PERMUTE", "EAAS_ENTRY_FFN_GROUPED",
    "EAAS_ENTRY_FORWARD", "eaas_expert_forward_noalloc", "EAAS_NOALLOC_SCRATCH_BYTES",
    "use_library", "EAAS_FP8_E4M3_TILED", "EAAS_GATE_UP", "EAAS_DOWN", "eaas_tile_weights_fp8",
]

EAAS_OK = 0
EAAS_BF16, EAAS_FP8_E4M3, EAAS_FP32, EAAS_FP8_E4M3_A8, EAAS_FP8_E4M3_TILED = 0, 1, 2, 3, 4
EAAS_GATE_UP, EAAS_DOWN = 0, 1
EAAS_SLOT_EMPTY, EAAS_SLOT_READY, EAAS_SLOT_DONE, EAAS_SLOT_OFFLINE = 0, 1, 2, 3
EAAS_WS_H, EAAS_WS_HQ, EAAS_WS_HS, EAAS_WS_XQ, EAAS_WS_XS, EAAS_WS_STAGE = range(6)
EAAS_ENTRY_ROUTE_PERMUTE, EAAS_ENTRY_FFN_GROUPED, EAAS_ENTRY_FORWARD = range(3)
EAAS_NOALLOC_SCRATCH_BYTES = 80 << 20
EXPORTED = ("eaas_workspace_bytes", "eaas_route_permute", "eaas_expert_ffn_grouped",
            "eaas_unpermute_combine", "eaas_expert_forward", "eaas_expert_forward_profiled",
            "eaas_status_string", "eaas_segments_workspace_bytes",
            "eaas_expert_forward_segments", "eaas_server_workspace_bytes", "eaas_server_step",
            "eaas_quantize_rows_fp8", "eaas_workspace_region", "eaas_workspace_bytes_for",
            "eaas_expert_forward_noalloc", "eaas_tile_weights_fp8")

_DEFAULT_LIB = Path(__file__).resolve().parent / "libeaas.so"
_LIB_PATH = _DEFAULT_LIB
_lib = None


class EaasError(RuntimeError):
    def __init__(self, status: int, where: str):
        super().__init__(f"{where}: {eaas_status_string(status)} (status {status})")
        self.status = status


class _Shape(ctypes.Structure):
    _fields_ = [("T", ctypes.c_int32), ("H", ctypes.c_int32), ("I", ctypes.c_int32),
                ("E", ctypes.c_int32), ("k", ctypes.c_int32)]


class _Routing(ctypes.Structure):
    _fields_ = [("counts", ctypes.c_void_p), ("offsets", ctypes.c_void_p),
                ("perm", ctypes.c_void_p), ("inv", ctypes.c_void_p),
                ("active", ctypes.c_void_p)]


def library_path() -> Path:
    return _LIB_PATH


def _bind(L: ctypes.CDLL) -> ctypes.CDLL:
    vp, sz, i32 = ctypes.c_void_p, ctypes.c_size_t, ctypes.c_int
    sp, rp = ctypes.POINTER(_Shape), ctypes.POINTER(_Routing)
    L.eaas_workspace_bytes.argtypes = [sp, i32]
    L.eaas_workspace_bytes.restype = sz
    L.eaas_workspace_bytes_for.argtypes = [sp, i32, i32]
    L.eaas_workspace_bytes_for.restype = sz
    L.eaas_route_permute.argtypes = [sp, vp, rp, vp, sz, vp]
    L.eaas_route_permute.restype = i32
    L.eaas_expert_ffn_grouped.argtypes = [sp, vp, rp, vp, vp, vp, vp, i32, vp, vp, sz, vp]
    L.eaas_expert_ffn_grouped.restype = i32
    L.eaas_unpermute_combine.argtypes = [sp, vp, rp, vp, vp, i32, vp]
    L.eaas_unpermute_combine.restype = i32
    L.eaas_expert_forward.argtypes = [sp, vp, vp, vp, vp, vp, vp, vp, i32, vp, i32, rp, vp, sz, vp]
    L.eaas_expert_forward.restype = i32
    L.eaas_expert_forward_profiled.argtypes = [sp, vp, vp, vp, vp, vp, vp, vp, i32, vp, i32,
                                               rp, vp, sz, vp, vp]
    L.eaas_expert_forward_profiled.restype = i32
    L.eaas_expert_forward_noalloc.argtypes = [sp, vp, vp, vp, vp, vp, vp, vp, i32, vp, i32,
                                              rp, vp]
    L.eaas_expert_forward_noalloc.restype = i32
    L.eaas_segments_workspace_bytes.argtypes = [sp, i32]
    L.eaas_segments_workspace_bytes.restype = sz
    L.eaas_expert_forward_segments.argtypes = [sp, vp, vp, i32, vp, vp, vp, vp, i32, i32, vp,
                                               sz, vp]
    L.eaas_expert_forward_segments.restype = i32
    L.eaas_server_workspace_bytes.argtypes = [sp, i32, i32]
    L.eaas_server_workspace_bytes.restype = sz
    L.eaas_server_step.argtypes = [sp, vp, i32, vp, i32, i32, vp, sz, vp]
    L.eaas_server_step.restype = i32
    L.eaas_tile_weights_fp8.argtypes = [sp, i32, vp, vp, vp]
    L.eaas_tile_weights_fp8.restype = i32
    L.eaas_quantize_rows_fp8.argtypes = [vp, ctypes.c_int64, ctypes.c_int32, vp, vp, vp]
    L.eaas_quantize_rows_fp8.restype = i32
    L.eaas_workspace_region.argtypes = [sp, i32, i32, ctypes.POINTER(sz), ctypes.POINTER(sz)]
    L.eaas_workspace_region.restype = i32
    L.eaas_status_string.argtypes = [i32]
    L.eaas_status_string.restype = ctypes.c_char_p
    return L


def lib() -> ctypes.CDLL:
    """Load libeaas.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not _LIB_PATH.exists():
            raise RuntimeError(f"{_LIB_PATH} is missing: build it with __graft_entry__.build()")
        _lib = _bind(ctypes.CDLL(str(_LIB_PATH)))
    return _lib


def use_library(path) -> ctypes.CDLL:
    """Route every later call of this module through the library at `path`
    (a build of the same sources, e.g. a scheduler variant for the
    group-shrink ablation); None returns to libeaas.so."""
    global _lib, _LIB_PATH
    _LIB_PATH = Path(path) if path is not None else _DEFAULT_LIB
    _lib = None
    return lib()


def eaas_status_string(status: int) -> str:
    return lib().eaas_status_string(int(status)).decode()


def _shape(T, H, I, E, k) -> _Shape:
    return _Shape(int(T), int(H), int(I), int(E), int(k))


def _p(t):
    if t is None:
        return None
    if isinstance(t, int):
        return t
    if not t.is_contiguous():
        raise ValueError("tensor arguments must be contiguous")
    return t.data_ptr()


def _stream(stream):
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


def _routing(r) -> _Routing | None:
    if r is None:
        return None
    return _Routing(_p(r["counts"]), _p(r["offsets"]), _p(r["perm"]), _p(r["inv"]), _p(r["active"]))


def _check(status: int, where: str) -> None:
    if status != EAAS_OK:
        raise EaasError(status, where)


def _wdtype(w: torch.Tensor, act8: bool = False, tiled: bool = False) -> int:
    if w.element_size() == 1:
        if act8 and tiled:
            raise ValueError("the tiled weight layout is for fp8 weights with bf16 activations")
        return EAAS_FP8_E4M3_A8 if act8 else (EAAS_FP8_E4M3_TILED if tiled else EAAS_FP8_E4M3)
    if act8 or tiled:
        raise ValueError("fp8 activations and the tiled layout need fp8-e4m3 (1-byte) weights")
    if w.element_size() == 2:
        return EAAS_BF16
    raise ValueError("weights must be bf16 (2-byte) or fp8-e4m3 (1-byte) tensors")


def eaas_workspace_region(T, H, I, E, k, w_dtype, region) -> tuple[int, int]:
    """(byte offset, bytes) of an intermediate inside the workspace."""
    s = _shape(T, H, I, E, k)
    off, n = ctypes.c_size_t(), ctypes.c_size_t()
    _check(lib().eaas_workspace_region(ctypes.byref(s), int(w_dtype), int(region),
                                       ctypes.byref(off), ctypes.byref(n)), "eaas_workspace_region")
    return off.value, n.value


def workspace_view(ws: torch.Tensor, T, H, I, E, k, w_dtype, region) -> torch.Tensor:
    """The bytes of one workspace region, as a uint8 view of `ws`."""
    off, n = eaas_workspace_region(T, H, I, E, k, w_dtype, region)
    return ws[off: off + n]


def eaas_quantize_rows_fp8(x: torch.Tensor, q: torch.Tensor, s: torch.Tensor, stream=None) -> None:
    """x [rows, K] bf16 -> q [rows, K] e4m3fn codes (uint8), s [rows, K/128] fp32."""
    rows, K = x.shape
    _check(lib().eaas_quantize_rows_fp8(_p(x), rows, K, _p(q), _p(s), _stream(stream)),
           "eaas_quantize_rows_fp8")


def eaas_tile_weights_fp8(w: torch.Tensor, which: int, H: int, I: int, out: torch.Tensor,
                          stream=None) -> None:
    """fp8 weights [E,N,K] (which = EAAS_GATE_UP: N = 2I, K = H; EAAS_DOWN:
    N = H, K = I) -> `out`, the same bytes in the tiled layout of
    EAAS_FP8_E4M3_TILED."""
    E = w.shape[0]
    s = _shape(0, H, I, E, 1)
    if out.numel() * out.element_size() != w.numel() * w.element_size():
        raise ValueError("out must hold as many bytes as w")
    _check(lib().eaas_tile_weights_fp8(ctypes.byref(s), int(which), _p(w), _p(out), _stream(stream)),
           "eaas_tile_weights_fp8")


def eaas_workspace_bytes(T, H, I, E, k, w_dtype=EAAS_BF16) -> int:
    s = _shape(T, H, I, E, k)
    return int(lib().eaas_workspace_bytes(ctypes.byref(s), int(w_dtype)))


def eaas_workspace_bytes_for(T, H, I, E, k, w_dtype, entry) -> int:
    s = _shape(T, H, I, E, k)
    return int(lib().eaas_workspace_bytes_for(ctypes.byref(s), int(w_dtype), int(entry)))


def alloc_workspace(T, H, I, E, k, w_dtype=EAAS_BF16, device="cuda") -> torch.Tensor:
    n = eaas_workspace_bytes(T, H, I, E, k, w_dtype)
    if n == 0:
        raise EaasError(-2, "eaas_workspace_bytes")
    return torch.empty(n, dtype=torch.uint8, device=device)


def alloc_routing(T, k, E, device="cuda") -> dict:
    R = T * k
    z = lambda n: torch.empty(max(n, 1), dtype=torch.int32, device=device)  # noqa: E731
    return dict(counts=z(E), offsets=z(E + 1), perm=z(R), inv=z(R), active=z(E + 1))


def eaas_route_permute(topk_ids: torch.Tensor, E: int, routing: dict, ws: torch.Tensor,
                       H: int = 128, I: int = 128, stream=None) -> None:
    T, k = topk_ids.shape
    s = _shape(T, H, I, E, k)
    r = _routing(routing)
    st = lib().eaas_route_permute(ctypes.byref(s), _p(topk_ids), ctypes.byref(r), _p(ws),
                                  ws.numel(), _stream(stream))
    _check(st, "eaas_route_permute")


def eaas_expert_ffn_grouped(x: torch.Tensor, routing: dict, w_gate_up: torch.Tensor,
                            w_down: torch.Tensor, y_perm: torch.Tensor, ws: torch.Tensor,
                            k: int, w_gate_up_scale=None, w_down_scale=None, stream=None,
                            act8: bool = False, tiled: bool = False) -> None:
    T, H = x.shape
    E, twoI, _ = w_gate_up.shape
    s = _shape(T, H, twoI // 2, E, k)
    r = _routing(routing)
    st = lib().eaas_expert_ffn_grouped(
        ctypes.byref(s), _p(x), ctypes.byref(r), _p(w_gate_up), _p(w_gate_up_scale),
        _p(w_down), _p(w_down_scale), _wdtype(w_gate_up, act8, tiled), _p(y_perm), _p(ws),
        ws.numel(), _stream(stream))
    _check(st, "eaas_expert_ffn_grouped")


def eaas_unpermute_combine(y_perm: torch.Tensor, routing: dict, topk_weights: torch.Tensor,
                           out: torch.Tensor, E: int, I: int = 128, stream=None) -> None:
    T, k = topk_weights.shape
    H = out.shape[1]
    s = _shape(T, H, I, E, k)
    r = _routing(routing)
    odt = EAAS_FP32 if out.dtype == torch.float32 else EAAS_BF16
    st = lib().eaas_unpermute_combine(ctypes.byref(s), _p(y_perm), ctypes.byref(r),
                                      _p(topk_weights), _p(out), odt, _stream(stream))
    _check(st, "eaas_unpermute_combine")


def eaas_expert_forward(x: torch.Tensor, topk_ids: torch.Tensor, topk_weights: torch.Tensor,
                        w_gate_up: torch.Tensor, w_down: torch.Tensor, out: torch.Tensor,
                        ws: torch.Tensor, w_gate_up_scale=None, w_down_scale=None,
                        routing: dict | None = None, stream=None, events=None,
                        act8: bool = False, tiled: bool = False) -> None:
    """events: optional 5 torch.cuda.Event(enable_timing=True) recorded on the
    stream around routing, gate/up, down and combine (profiled entry point).
    act8: fp8 activations with the fp8 weights (EAAS_FP8_E4M3_A8).
    tiled: the fp8 weights are in the layout of eaas_tile_weights_fp8."""
    T, H = x.shape
    E, twoI, _ = w_gate_up.shape
    k = topk_ids.shape[1]
    s = _shape(T, H, twoI // 2, E, k)
    r = _routing(routing)
    odt = EAAS_FP32 if out.dtype == torch.float32 else EAAS_BF16
    args = (ctypes.byref(s), _p(x), _p(topk_ids), _p(topk_weights), _p(w_gate_up),
            _p(w_gate_up_scale), _p(w_down), _p(w_down_scale), _wdtype(w_gate_up, act8, tiled),
            _p(out), odt, ctypes.byref(r) if r is not None else None, _p(ws), ws.numel(),
            _stream(stream))
    if events is None:
        _check(lib().eaas_expert_forward(*args), "eaas_expert_forward")
        return
    if len(events) != 5:
        raise ValueError("events must hold 5 entries")
    ev = (ctypes.c_void_p * 5)(*[e.cuda_event if e is not None else None for e in events])
    _check(lib().eaas_expert_forward_profiled(*args, ev), "eaas_expert_forward_profiled")


def eaas_expert_forward_noalloc(x: torch.Tensor, topk_ids: torch.Tensor,
                                topk_weights: torch.Tensor, w_gate_up: torch.Tensor,
                                w_down: torch.Tensor, out: torch.Tensor, w_gate_up_scale=None,
                                w_down_scale=None, routing: dict | None = None, stream=None,
                                act8: bool = False, tiled: bool = False) -> None:
    """eaas_expert_forward on the library's own per-GPU scratch array: no
    workspace argument, nothing allocated (shapes up to
    EAAS_NOALLOC_SCRATCH_BYTES of workspace)."""
    T, H = x.shape
    E, twoI, _ = w_gate_up.shape
    k = topk_ids.shape[1]
    s = _shape(T, H, twoI // 2, E, k)
    r = _routing(routing)
    odt = EAAS_FP32 if out.dtype == torch.float32 else EAAS_BF16
    _check(lib().eaas_expert_forward_noalloc(
        ctypes.byref(s), _p(x), _p(topk_ids), _p(topk_weights), _p(w_gate_up),
        _p(w_gate_up_scale), _p(w_down), _p(w_down_scale), _wdtype(w_gate_up, act8, tiled), _p(out),
        odt, ctypes.byref(r) if r is not None else None, _stream(stream)),
        "eaas_expert_forward_noalloc")


def eaas_expert_forward_profiled(*args, events, **kwargs) -> None:
    """eaas_expert_forward with timing events (see eaas_expert_forward)."""
    for e in events:
        if e is not None and not e.cuda_event:
            e.record()  # torch creates the underlying HIP event lazily
    eaas_expert_forward(*args, events=events, **kwargs)


# ------------------------------------------------------------ dynamic batch
def eaas_segments_workspace_bytes(T, H, I, E, k, w_dtype=EAAS_BF16) -> int:
    s = _shape(T, H, I, E, k)
    return int(lib().eaas_segments_workspace_bytes(ctypes.byref(s), int(w_dtype)))


def alloc_segments_workspace(T, H, I, E, k, w_dtype=EAAS_BF16, device="cuda") -> torch.Tensor:
    n = eaas_segments_workspace_bytes(T, H, I, E, k, w_dtype)
    if n == 0:
        raise EaasError(-2, "eaas_segments_workspace_bytes")
    return torch.empty(n, dtype=torch.uint8, device=device)


def segment_table(segments, device="cuda") -> torch.Tensor:
    """Device array of eaas_segment records ([n, 4] int64: x, topk_ids,
    topk_weights, out pointers) for a list of (x, topk_ids, topk_weights, out)
    tensors.  Build it once per set of buffers; the token counts are passed
    separately, so the same table serves every step."""
    rows = [[_p(x), _p(ids), _p(w), _p(out)] for (x, ids, w, out) in segments]
    t = torch.tensor(rows if rows else [[0, 0, 0, 0]], dtype=torch.int64)
    return t.to(device)


def eaas_expert_forward_segments(table: torch.Tensor, num_tokens: torch.Tensor, n_seg: int,
                                 capacity: int, k: int, w_gate_up: torch.Tensor,
                                 w_down: torch.Tensor, ws: torch.Tensor, out_dtype=EAAS_BF16,
                                 w_gate_up_scale=None, w_down_scale=None, stream=None,
                                 act8: bool = False, tiled: bool = False) -> None:
    """The step on a dynamic batch: `table` from segment_table, `num_tokens`
    a device int32 tensor of the requests' token counts (read on the device),
    `capacity` the bound on their sum.  act8: fp8 activations."""
    E, twoI, H = w_gate_up.shape
    s = _shape(capacity, H, twoI // 2, E, k)
    st = lib().eaas_expert_forward_segments(
        ctypes.byref(s), _p(table), _p(num_tokens), int(n_seg), _p(w_gate_up),
        _p(w_gate_up_scale), _p(w_down), _p(w_down_scale), _wdtype(w_gate_up, act8, tiled),
        int(out_dtype), _p(ws), ws.numel(), _stream(stream))
    _check(st, "eaas_expert_forward_segments")


# ------------------------------------------------------------ server step
def eaas_server_workspace_bytes(T, H, I, E, k, n_layers, w_dtype=EAAS_BF16) -> int:
    s = _shape(T, H, I, E, k)
    return int(lib().eaas_server_workspace_bytes(ctypes.byref(s), int(n_layers), int(w_dtype)))


def alloc_server_workspace(T, H, I, E, k, n_layers, w_dtype=EAAS_BF16,
                           device="cuda") -> torch.Tensor:
    n = eaas_server_workspace_bytes(T, H, I, E, k, n_layers, w_dtype)
    if n == 0:
        raise EaasError(-2, "eaas_server_workspace_bytes")
    return torch.empty(n, dtype=torch.uint8, device=device)


def slot_table(slots, device="cuda") -> torch.Tensor:
    """Device array of eaas_slot records ([n, 6] int64) for a list of
    (flag, header, x, topk_ids, topk_weights) device tensors; the capacity is
    x's row count."""
    rows = [[_p(f), _p(h), _p(x), _p(i), _p(w), int(x.shape[0])] for (f, h, x, i, w) in slots]
    t = torch.tensor(rows if rows else [[0] * 6], dtype=torch.int64)
    return t.to(device)


def layer_table(layers, device="cuda") -> torch.Tensor:
    """Device array of eaas_layer_weights records ([n, 4] int64) for a list of
    (w_gate_up, w_gate_up_scale, w_down, w_down_scale) tensors (scales None
    for bf16 weights)."""
    rows = [[_p(a) or 0, _p(b) or 0, _p(c) or 0, _p(d) or 0] for (a, b, c, d) in layers]
    return torch.tensor(rows, dtype=torch.int64).to(device)


def eaas_server_step(slots: torch.Tensor, n_slots: int, layers: torch.Tensor, n_layers: int,
                     capacity: int, H: int, I: int, E: int, k: int, ws: torch.Tensor,
                     w_dtype=EAAS_BF16, stream=None) -> None:
    """One server step over the slots of `slot_table` with the weights of
    `layer_table` (E experts per layer)."""
    s = _shape(capacity, H, I, E, k)
    st = lib().eaas_server_step(ctypes.byref(s), _p(slots), int(n_slots), _p(layers),
                                int(n_layers), int(w_dtype), _p(ws), ws.numel(), _stream(stream))
    _check(st, "eaas_server_step")
