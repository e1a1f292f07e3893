"""Chunked scan on the GPU (through the C ABI) against the CPU oracle.

Parity bar: max |x - y| / max |y| <= 2e-3 per output tensor (o, every chunk
state, the final state), bf16 (or fp32) inputs and fp32 state against the
fp64 oracle.  GPU-vs-GPU continuation at chunk-aligned boundaries is bitwise.
"""
import numpy as np
import pytest

import paper_2606_20537_amd as cap
from gpu_util import PARITY_TOL, SPLIT_TOL, dev_inputs, rel_err, scan_case

pytestmark = pytest.mark.gpu


def _run(inp, T, H, dk, dv, S0=None, want_cs=True, want_final=True, scale=1.0):
    import torch
    d = dev_inputs(inp)
    n_chunks = (T + 63) // 64
    o = torch.full((T, H, dv), float("nan"), dtype=torch.float32, device="cuda")
    cs = torch.full((n_chunks, H, dk, dv), float("nan"), dtype=torch.float32, device="cuda") if want_cs else None
    fs = torch.full((H, dk, dv), float("nan"), dtype=torch.float32, device="cuda") if want_final else None
    s_in = torch.from_numpy(S0.astype(np.float32)).cuda() if S0 is not None else None
    cap.linattn_chunked_prefill(d["q"], d["k"], d["v"], d["g"], o, state_in=s_in, chunk_states=cs,
                                final_state=fs, T=T, H=H, dk=dk, dv=dv, scale=scale,
                                in_dtype=cap.CAP_DTYPE_F32 if d["q"].dtype == torch.float32 else cap.CAP_DTYPE_BF16)
    torch.cuda.synchronize()
    return (o.cpu().numpy(), None if cs is None else cs.cpu().numpy(), None if fs is None else fs.cpu().numpy())


CASES = [
    # (id, T, H, dk, dv, dtype, with_S0)
    ("tiny_f32", 256, 2, 64, 64, "f32", False),
    ("f32_ragged_state", 150, 2, 64, 32, "f32", True),
    ("bf16_dk128_ragged_oddH", 200, 3, 128, 32, "bf16", True),
    ("bf16_dk64_xcd_map", 130, 8, 64, 64, "bf16", False),
    ("bf16_dv16", 97, 4, 128, 16, "bf16", True),
    ("bf16_hybrid8_layer", 2048, 16, 128, 128, "bf16", False),
    ("bf16_one_chunk_exact", 64, 2, 128, 128, "bf16", True),
    ("bf16_one_token", 1, 2, 128, 128, "bf16", True),
    ("bf16_one_token_dk64_oddH", 1, 3, 64, 48, "bf16", True),
    ("bf16_one_token_zero_state", 1, 5, 128, 16, "bf16", False),
    ("f32_one_token", 1, 2, 64, 64, "f32", True),
    ("bf16_63", 63, 2, 128, 48, "bf16", True),
    ("bf16_65", 65, 2, 128, 48, "bf16", True),
    # 16 slices per head, 512 workgroups: more than one workgroup per CU over the call
    ("bf16_dv256_512_workgroups", 200, 32, 128, 256, "bf16", True),
]


@pytest.mark.parametrize("cid,T,H,dk,dv,dtype,with_s0", CASES, ids=[c[0] for c in CASES])
def test_scan_parity(orc, cid, T, H, dk, dv, dtype, with_s0):
    print("case", cid, T, H, dk, dv, dtype, flush=True)
    inp = scan_case(100 + T + H, T, H, dk, dv, dtype)
    S0 = None
    if with_s0:
        S0 = np.random.default_rng(T).standard_normal((H, dk, dv)).astype(np.float32)
    o, cs, fs = _run(inp, T, H, dk, dv, S0=S0)
    o_ref, S_ref = orc.sequential(inp["q"], inp["k"], inp["v"], inp["g"], S0=S0)
    _, cs_ref, _ = orc.chunked(inp["q"], inp["k"], inp["v"], inp["g"], 64, S0=S0)
    e_o, e_s = rel_err(o, o_ref), rel_err(fs, S_ref)
    e_cs = max(rel_err(cs[j], cs_ref[j]) for j in range(cs.shape[0]))
    print("  rel err o %.3g final %.3g chunk states %.3g" % (e_o, e_s, e_cs), flush=True)
    assert np.all(np.isfinite(o)) and np.all(np.isfinite(cs)) and np.all(np.isfinite(fs))
    assert e_o <= PARITY_TOL and e_s <= PARITY_TOL and e_cs <= PARITY_TOL
    # the hi/lo operand split is designed for ~1e-5; a dropped lo term shows up here
    assert e_o <= SPLIT_TOL and e_s <= SPLIT_TOL and e_cs <= SPLIT_TOL


def test_scan_zero_length(orc):
    """T = 0: nothing but final_state = state_in."""
    H, dk, dv = 2, 128, 32
    inp = scan_case(7, 0, H, dk, dv)
    S0 = np.random.default_rng(1).standard_normal((H, dk, dv)).astype(np.float32)
    o, cs, fs = _run(inp, 0, H, dk, dv, S0=S0)
    assert np.array_equal(fs, S0)


def test_scan_gate_extremes(orc):
    """g = -100 (state wiped every token) and g = 0 (no decay)."""
    T, H, dk, dv = 130, 2, 128, 32
    for gv in (-100.0, 0.0):
        inp = scan_case(11, T, H, dk, dv)
        inp["g"][:] = np.float32(gv)
        o, cs, fs = _run(inp, T, H, dk, dv)
        o_ref, S_ref = orc.sequential(inp["q"], inp["k"], inp["v"], inp["g"])
        assert rel_err(o, o_ref) <= SPLIT_TOL and rel_err(fs, S_ref) <= SPLIT_TOL, gv


def test_scan_optional_outputs_and_inplace(orc):
    """chunk_states / final_state may be NULL; final_state may alias state_in;
    none of this changes o by a single bit."""
    import torch
    T, H, dk, dv = 150, 4, 128, 64
    inp = scan_case(13, T, H, dk, dv)
    S0 = np.random.default_rng(2).standard_normal((H, dk, dv)).astype(np.float32)
    o_a, cs_a, fs_a = _run(inp, T, H, dk, dv, S0=S0)
    o_b, _, _ = _run(inp, T, H, dk, dv, S0=S0, want_cs=False, want_final=False)
    assert np.array_equal(o_a, o_b)
    d = dev_inputs(inp)
    st = torch.from_numpy(S0).cuda()
    o = torch.empty((T, H, dv), dtype=torch.float32, device="cuda")
    cap.linattn_chunked_prefill(d["q"], d["k"], d["v"], d["g"], o, state_in=st, final_state=st)
    torch.cuda.synchronize()
    assert np.array_equal(o.cpu().numpy(), o_a) and np.array_equal(st.cpu().numpy(), fs_a)


def test_scan_scale(orc):
    T, H, dk, dv = 100, 2, 64, 32
    inp = scan_case(17, T, H, dk, dv)
    o1, _, _ = _run(inp, T, H, dk, dv, scale=1.0)
    o2, _, _ = _run(inp, T, H, dk, dv, scale=0.125)
    assert np.array_equal(o2, 0.125 * o1)


def test_scan_deterministic():
    """Two runs give identical bits (no atomics, fixed reduction order)."""
    T, H, dk, dv = 700, 16, 128, 128
    inp = scan_case(19, T, H, dk, dv)
    a = _run(inp, T, H, dk, dv)
    b = _run(inp, T, H, dk, dv)
    for x, y in zip(a, b):
        assert np.array_equal(x, y)


@pytest.mark.parametrize("P", [0, 64, 128, 640, 1984])
def test_aligned_continuation_bitwise(P):
    """Prefill [0, F) in one call equals prefill [0, P) then [P, F) from the
    handed-over state, bit for bit, when P is a multiple of the chunk (§5)."""
    import torch
    T, H, dk, dv = 2048, 16, 128, 128
    inp = scan_case(23, T, H, dk, dv)
    d = dev_inputs(inp)
    o_full = torch.empty((T, H, dv), dtype=torch.float32, device="cuda")
    cs_full = torch.empty(((T + 63) // 64, H, dk, dv), dtype=torch.float32, device="cuda")
    fs_full = torch.empty((H, dk, dv), dtype=torch.float32, device="cuda")
    cap.linattn_chunked_prefill(d["q"], d["k"], d["v"], d["g"], o_full, chunk_states=cs_full, final_state=fs_full)
    o_a = torch.empty((P, H, dv), dtype=torch.float32, device="cuda")
    st = torch.empty((H, dk, dv), dtype=torch.float32, device="cuda")
    cap.linattn_chunked_prefill(d["q"][:P], d["k"][:P], d["v"][:P], d["g"][:P], o_a, final_state=st,
                                T=P, H=H, dk=dk, dv=dv, in_dtype=cap.CAP_DTYPE_BF16)
    st_P = st.clone()
    o_b = torch.empty((T - P, H, dv), dtype=torch.float32, device="cuda")
    cap.linattn_chunked_prefill(d["q"][P:], d["k"][P:], d["v"][P:], d["g"][P:], o_b, state_in=st, final_state=st,
                                T=T - P, H=H, dk=dk, dv=dv, in_dtype=cap.CAP_DTYPE_BF16)
    torch.cuda.synchronize()
    assert torch.equal(torch.cat([o_a, o_b]), o_full)
    assert torch.equal(st, fs_full)
    # the chunk-boundary state output at P is the state a prefill stopping at P hands over
    assert torch.equal(st_P, cs_full[P // 64])


@pytest.mark.parametrize("dk,dv", [(128, 128), (64, 32)])
def test_one_token_state_equals_chunked_fold(dk, dv):
    """A one-token prefill from a chunk boundary is the chunked kernel's
    one-token chunk: token 64 of one 65-token call against a one-token call
    from that call's chunk-boundary state 1 -- o and the state equal bit for
    bit.  The decode step (vector-ALU path) folds the state bit-identically
    and agrees on o to fp32 rounding."""
    import torch
    T, H = 65, 4
    inp = scan_case(41, T, H, dk, dv)
    S0 = np.random.default_rng(7).standard_normal((H, dk, dv)).astype(np.float32)
    o, cs, fs = _run(inp, T, H, dk, dv, S0=S0)
    d = dev_inputs(inp)
    st = torch.from_numpy(cs[1]).cuda()
    o1 = torch.empty((1, H, dv), dtype=torch.float32, device="cuda")
    cs1 = torch.empty((1, H, dk, dv), dtype=torch.float32, device="cuda")
    fs1 = torch.empty((H, dk, dv), dtype=torch.float32, device="cuda")
    cap.linattn_chunked_prefill(d["q"][64:], d["k"][64:], d["v"][64:], d["g"][64:], o1, state_in=st,
                                chunk_states=cs1, final_state=fs1, T=1, H=H, dk=dk, dv=dv,
                                in_dtype=cap.CAP_DTYPE_BF16)
    o2 = torch.empty((1, H, dv), dtype=torch.float32, device="cuda")
    fs2 = torch.empty((H, dk, dv), dtype=torch.float32, device="cuda")
    cap.linattn_decode_step(d["q"][64:], d["k"][64:], d["v"][64:], d["g"][64:], o2, state_in=st,
                            final_state=fs2, T=1, H=H, dk=dk, dv=dv, in_dtype=cap.CAP_DTYPE_BF16)
    torch.cuda.synchronize()
    assert np.array_equal(fs1.cpu().numpy(), fs)
    assert np.array_equal(cs1.cpu().numpy()[0], cs[1])  # entry 0 is the state entering the call
    assert np.array_equal(o1.cpu().numpy()[0], o[64])
    assert np.array_equal(fs2.cpu().numpy(), fs)
    assert rel_err(o2.cpu().numpy()[0], o[64]) <= SPLIT_TOL


def test_decode_step_argument_checks():
    """The decode step takes exactly one token."""
    import torch
    H, dk, dv = 2, 128, 16
    inp = scan_case(45, 2, H, dk, dv)
    d = dev_inputs(inp)
    o = torch.empty((2, H, dv), dtype=torch.float32, device="cuda")
    for T in (0, 2):
        with pytest.raises(cap.CapsuleError) as ei:
            cap.linattn_decode_step(d["q"], d["k"], d["v"], d["g"], o, T=T, H=H, dk=dk, dv=dv)
        assert ei.value.status == cap.CAP_E_UNSUPPORTED


def test_one_token_inplace_and_optional_outputs(orc):
    """One-token calls: final_state may be state_in; chunk_states / final_state
    may be NULL; a NULL state_in is the zero state."""
    import torch
    H, dk, dv = 3, 128, 64
    inp = scan_case(43, 1, H, dk, dv)
    S0 = np.random.default_rng(9).standard_normal((H, dk, dv)).astype(np.float32)
    o_a, cs_a, fs_a = _run(inp, 1, H, dk, dv, S0=S0)
    o_b, _, _ = _run(inp, 1, H, dk, dv, S0=S0, want_cs=False, want_final=False)
    assert np.array_equal(o_a, o_b) and np.array_equal(cs_a[0], S0)
    d = dev_inputs(inp)
    st = torch.from_numpy(S0).cuda()
    o = torch.empty((1, H, dv), dtype=torch.float32, device="cuda")
    cap.linattn_chunked_prefill(d["q"], d["k"], d["v"], d["g"], o, state_in=st, final_state=st)
    torch.cuda.synchronize()
    assert np.array_equal(o.cpu().numpy(), o_a) and np.array_equal(st.cpu().numpy(), fs_a)
    # the decode step in place: the same state bits, o to fp32 rounding
    st2 = torch.from_numpy(S0).cuda()
    o2 = torch.empty((1, H, dv), dtype=torch.float32, device="cuda")
    cap.linattn_decode_step(d["q"], d["k"], d["v"], d["g"], o2, state_in=st2, final_state=st2)
    torch.cuda.synchronize()
    assert np.array_equal(st2.cpu().numpy(), fs_a) and rel_err(o2.cpu().numpy(), o_a) <= SPLIT_TOL
    o_z, cs_z, fs_z = _run(inp, 1, H, dk, dv)
    o_ref, s_ref = orc.sequential(inp["q"], inp["k"], inp["v"], inp["g"])
    assert not cs_z.any() and rel_err(o_z, o_ref) <= SPLIT_TOL and rel_err(fs_z, s_ref) <= SPLIT_TOL
