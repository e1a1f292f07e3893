"""Helpers shared by the GPU tests (device placement, comparison metrics).

Inputs come from ``synth`` and expected values from ``oracle``; nothing here
computes any part of the method."""
import os
from concurrent.futures import ThreadPoolExecutor

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


def elem_err(x, y, floor=1e-3):
    """max_i |x_i - y_i| / max(|y_i|, floor * max|y|): the elementwise
    relative error with a magnitude floor (elements far below the tensor's
    scale are measured against the floor)."""
    x = np.asarray(x, np.float64)
    y = np.asarray(y, np.float64)
    if x.size == 0:
        return 0.0
    fl = floor * float(np.max(np.abs(y)))
    den = np.maximum(np.abs(y), fl)
    if fl == 0:
        den = np.where(den == 0, 1.0, den)
    return float(np.max(np.abs(x - y) / den))


def oracle_threads():
    """Worker threads for head-parallel oracle runs (the C oracle releases
    the GIL inside each call); at most 16, the CPU share of one GPU."""
    return max(1, min(16, len(os.sched_getaffinity(0))))


def by_head(fn, arrays, heads):
    """Run an oracle function on each head h of ``heads`` separately (arrays
    sliced [:, h:h+1] along the head axis, made contiguous) in worker
    threads; returns the list of per-head results, in order."""
    def one(h):
        return fn(*[np.ascontiguousarray(a[:, h:h + 1]) for a in arrays])
    with ThreadPoolExecutor(oracle_threads()) as ex:
        return list(ex.map(one, heads))


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
