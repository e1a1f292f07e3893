"""Helpers shared by the GPU tests (device placement, comparison metrics).

Inputs come from ``synth`` and expected values from ``oracle``; nothing here
computes any part of the method."""
import numpy as np

import synth

PARITY_TOL = 2e-3     # max |x - y| / max |y| per output tensor (bf16 in, fp32 state)
SPLIT_TOL = 1e-4      # what the hi/lo bf16 operand split is expected to reach


def torch_mod():
    import torch
    return torch


def dev_inputs(inp):
    """Device tensors for synth.linattn_inputs output (bf16 or fp32 payloads)."""
    torch = torch_mod()
    out = {}
    for name in ("q", "k", "v"):
        pay = inp[name + "_dev"]
        if pay.dtype == np.uint16:
            t = torch.from_numpy(pay.view(np.int16).copy()).view(torch.bfloat16)
        else:
            t = torch.from_numpy(np.ascontiguousarray(pay))
        out[name] = t.cuda().contiguous()
    out["g"] = torch.from_numpy(inp["g"]).cuda().contiguous()
    return out


def rel_err(x, y):
    """max |x - y| / max |y| (the parity metric)."""
    x = np.asarray(x, np.float64)
    y = np.asarray(y, np.float64)
    if x.size == 0:
        return 0.0
    den = float(np.max(np.abs(y)))
    num = float(np.max(np.abs(x - y)))
    return num / den if den > 0 else num


def scan_case(seed, T, H, dk, dv, dtype="bf16", gate_mu=3.0, gate_sigma=0.5):
    return synth.linattn_inputs(seed, 0, T, H, dk, dv, dtype, gate_mu=gate_mu, gate_sigma=gate_sigma)


def device_bytes(nbytes, fill=None, seed=None, name="buf"):
    """uint8 device buffer: random N(0,1) float32 payload (seeded) or a fill byte."""
    torch = torch_mod()
    if seed is not None:
        host = synth.fill_normal_bytes(seed, 0, name, nbytes)
        return torch.from_numpy(host.copy()).cuda()
    t = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    t.fill_(0 if fill is None else fill)
    return t
