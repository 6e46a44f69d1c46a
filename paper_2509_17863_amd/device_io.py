"""Copy seeded host inputs (numpy bit patterns) into device tensors."""
from __future__ import annotations

import numpy as np
import torch


def _bf16(a: np.ndarray, device) -> torch.Tensor:
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(device)


def to_device(inp: dict, device="cuda") -> dict:
    """Device tensors for the binding: x bf16 [T,H], topk_ids int32, topk_weights
    fp32, weights bf16 or fp8-e4m3 (uint8 bits viewed as float8_e4m3fn), scales fp32."""
    d = dict(x=_bf16(inp["x"], device),
             topk_ids=torch.from_numpy(np.ascontiguousarray(inp["topk_ids"])).to(device),
             topk_weights=torch.from_numpy(np.ascontiguousarray(inp["topk_weights"])).to(device))
    if inp["wdtype"] == "bf16":
        d["w_gate_up"] = _bf16(inp["w_gate_up"], device)
        d["w_down"] = _bf16(inp["w_down"], device)
        d["w_gate_up_scale"] = d["w_down_scale"] = None
    else:
        d["w_gate_up"] = torch.from_numpy(inp["w_gate_up"]).to(device).view(torch.float8_e4m3fn)
        d["w_down"] = torch.from_numpy(inp["w_down"]).to(device).view(torch.float8_e4m3fn)
        d["w_gate_up_scale"] = torch.from_numpy(inp["w_gate_up_scale"]).to(device)
        d["w_down_scale"] = torch.from_numpy(inp["w_down_scale"]).to(device)
    return d


def bf16_tensor_to_bits(t: torch.Tensor) -> np.ndarray:
    return t.detach().cpu().contiguous().view(torch.int16).numpy().view(np.uint16)
