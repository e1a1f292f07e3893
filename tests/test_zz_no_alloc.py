"""gdn_chunked_prefill_noalloc -- the delta-rule prefill for callers that
cannot allocate -- against gdn_chunked_prefill with a caller workspace,
through the C ABI: bit-identical o, chunk states and final state on calls in
a row, the first long enough to run in several segments of the library's
fixed scratch, the next ones smaller (the scratch then holds the previous
call's contents)."""
import numpy as np
import pytest
import torch

import paper_2606_20537_amd as cap
import synth
from gpu_util import dev_inputs

pytestmark = pytest.mark.gpu


def _inputs(seed, T, H, dk, dv):
    inp = synth.gdn_inputs(seed, 0, T, H, dk, dv, "bf16")
    d = dev_inputs(inp)
    d["beta"] = torch.from_numpy(inp["beta"]).cuda()
    return d


def _outputs(T, H, dk, dv):
    n = (T + 63) // 64
    nan = float("nan")
    return (torch.full((T, H, dv), nan, device="cuda"), torch.full((n, H, dk, dv), nan, device="cuda"),
            torch.full((H, dk, dv), nan, device="cuda"))


def _segments(T, H, dk, dv):
    slot = -(-(H * dk * dv * 4) // 256) * 256
    per = (cap.GDN_NOALLOC_SCRATCH_BYTES - 2 * slot) // (H * 12800)
    return -(-((T + 63) // 64) // per)


def test_noalloc_equals_workspace_entry_point_on_calls_in_a_row():
    cases = [(16384 + 37, 32, 128, 128), (200, 4, 64, 32), (64, 2, 128, 16)]
    assert _segments(*cases[0]) >= 4 and _segments(*cases[1]) == 1
    gen = torch.Generator(device="cuda").manual_seed(77)
    for i, (T, H, dk, dv) in enumerate(cases):
        print("call %d: T %d H %d dk %d dv %d, %d segment(s)" % (i, T, H, dk, dv, _segments(T, H, dk, dv)),
              flush=True)
        d = _inputs(90 + i, T, H, dk, dv)
        s0 = torch.randn((H, dk, dv), generator=gen, device="cuda") * 0.1
        ref = _outputs(T, H, dk, dv)
        cap.gdn_chunked_prefill(d["q"], d["k"], d["v"], d["g"], d["beta"], ref[0], state_in=s0,
                                chunk_states=ref[1], final_state=ref[2])
        got = _outputs(T, H, dk, dv)
        cap.gdn_chunked_prefill_noalloc(d["q"], d["k"], d["v"], d["g"], d["beta"], got[0], state_in=s0,
                                        chunk_states=got[1], final_state=got[2])
        torch.cuda.synchronize()
        for name, x, y in zip(("o", "chunk states", "final state"), got, ref):
            assert torch.equal(x, y), (i, name)


def test_noalloc_inplace_state_optional_outputs_and_empty_call():
    """The state updated in place across segments, no chunk states, and a
    T = 0 call that only hands the entering state over."""
    T, H, dk, dv = 9000, 32, 128, 128
    assert _segments(T, H, dk, dv) >= 2
    d = _inputs(95, T, H, dk, dv)
    gen = torch.Generator(device="cuda").manual_seed(78)
    s0 = torch.randn((H, dk, dv), generator=gen, device="cuda") * 0.1
    o_ref = torch.empty((T, H, dv), device="cuda")
    st_ref = s0.clone()
    cap.gdn_chunked_prefill(d["q"], d["k"], d["v"], d["g"], d["beta"], o_ref, state_in=st_ref, final_state=st_ref)
    o = torch.empty((T, H, dv), device="cuda")
    st = s0.clone()
    cap.gdn_chunked_prefill_noalloc(d["q"], d["k"], d["v"], d["g"], d["beta"], o, state_in=st, final_state=st)
    fs0 = torch.full((H, dk, dv), float("nan"), device="cuda")
    cap.gdn_chunked_prefill_noalloc(None, None, None, None, None, None, state_in=s0, final_state=fs0,
                                    T=0, H=H, dk=dk, dv=dv)
    torch.cuda.synchronize()
    assert torch.equal(o, o_ref) and torch.equal(st, st_ref)
    assert torch.equal(fs0, s0)


def test_noalloc_rejections():
    T, H, dk, dv = 100, 2, 64, 16
    d = _inputs(96, T, H, dk, dv)
    o = torch.empty((T, H, dv), device="cuda")
    ws = torch.empty(cap.gdn_workspace_bytes(T, H), dtype=torch.uint8, device="cuda")
    import ctypes as ct
    from paper_2606_20537_amd import _native as N
    a = N.gdn_args(d["q"].data_ptr(), d["k"].data_ptr(), d["v"].data_ptr(), d["g"].data_ptr(),
                   d["beta"].data_ptr(), 0, o.data_ptr(), 0, 0, ws.data_ptr(), ws.numel(), T, H, dk, dv, 64,
                   cap.CAP_DTYPE_BF16, 1.0)
    assert N.load().gdn_chunked_prefill_noalloc(ct.byref(a), None) == cap.CAP_E_INVAL   # a workspace given
    o.fill_(float("nan"))
    torch.cuda.synchronize()
    assert torch.isnan(o).all()                                                          # nothing ran
    with pytest.raises(cap.CapsuleError) as ei:   # one chunk of 300 heads does not fit the scratch
        cap.gdn_chunked_prefill_noalloc(None, None, None, None, None, None, T=0, H=300, dk=128, dv=128)
    assert ei.value.status == cap.CAP_E_SIZE
