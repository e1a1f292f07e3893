"""Chunked gated delta-rule prefill on the GPU (through the C ABI) against the
CPU oracle.

Parity bar as for the linear-attention scan: max |x - y| / max |y| <= 2e-3
per output tensor (o, every chunk state, the final state) with bf16 inputs
and fp32 state against the fp64 oracle; GPU-vs-GPU continuation at
chunk-aligned boundaries is bitwise.  o and the final state are compared with
the token-by-token recurrence, the chunk states with the oracle's chunked
form."""
import numpy as np
import pytest

import paper_2606_20537_amd as cap
import synth
from gpu_util import PARITY_TOL, SPLIT_TOL, dev_inputs, rel_err

pytestmark = pytest.mark.gpu


def gdn_case(seed, T, H, dk, dv):
    return synth.gdn_inputs(seed, 0, T, H, dk, dv, "bf16")


def _dev(inp):
    import torch
    d = dev_inputs(inp)
    d["beta"] = torch.from_numpy(inp["beta"]).cuda().contiguous()
    return d


def _run(inp, T, H, dk, dv, S0=None, want_cs=True, want_final=True, scale=1.0):
    import torch
    d = _dev(inp)
    n_chunks = (T + 63) // 64
    o = torch.full((T, H, dv), float("nan"), dtype=torch.float32, device="cuda")
    cs = torch.full((n_chunks, H, dk, dv), float("nan"), dtype=torch.float32, device="cuda") if want_cs else None
    fs = torch.full((H, dk, dv), float("nan"), dtype=torch.float32, device="cuda") if want_final else None
    s_in = torch.from_numpy(S0.astype(np.float32)).cuda() if S0 is not None else None
    cap.gdn_chunked_prefill(d["q"], d["k"], d["v"], d["g"], d["beta"], o, state_in=s_in, chunk_states=cs,
                            final_state=fs, T=T, H=H, dk=dk, dv=dv, scale=scale)
    torch.cuda.synchronize()
    return (o.cpu().numpy(), None if cs is None else cs.cpu().numpy(), None if fs is None else fs.cpu().numpy())


def _refs(orc, inp, S0=None, scale=1.0):
    a = (inp["q"], inp["k"], inp["v"], inp["g"], inp["beta"])
    o_ref, s_ref = orc.gdn_sequential(*a, S0=S0, scale=scale)
    _, cs_ref, _ = orc.gdn_chunked(*a, 64, S0=S0, scale=scale)
    return o_ref, cs_ref, s_ref


CASES = [
    # (id, T, H, dk, dv, with_S0)
    ("dk64_two_heads", 256, 2, 64, 64, False),
    ("dk128_ragged_oddH", 200, 3, 128, 32, True),
    ("dk64_xcd_map", 130, 8, 64, 64, False),
    ("dv16", 97, 4, 128, 16, True),
    ("hybrid8_layer", 2048, 16, 128, 128, False),
    ("one_chunk_exact", 64, 2, 128, 128, True),
    ("one_token", 1, 2, 128, 128, True),
    ("one_token_dk64_oddH", 1, 3, 64, 48, True),
    ("one_token_zero_state", 1, 5, 128, 16, False),
    ("t63", 63, 2, 128, 48, True),
    ("t65", 65, 2, 128, 48, True),
    ("dk64_long", 1000, 2, 64, 32, True),
    # 512 workgroups: more than one workgroup per CU over the call
    ("h64_512_workgroups", 200, 64, 128, 128, True),
]


@pytest.mark.parametrize("cid,T,H,dk,dv,with_s0", CASES, ids=[c[0] for c in CASES])
def test_gdn_parity(orc, cid, T, H, dk, dv, with_s0):
    print("case", cid, T, H, dk, dv, flush=True)
    inp = gdn_case(200 + T + H, T, H, dk, dv)
    S0 = np.random.default_rng(T).standard_normal((H, dk, dv)).astype(np.float32) if with_s0 else None
    o, cs, fs = _run(inp, T, H, dk, dv, S0=S0)
    o_ref, cs_ref, s_ref = _refs(orc, inp, S0=S0)
    e_o, e_s = rel_err(o, o_ref), rel_err(fs, s_ref)
    e_cs = max(rel_err(cs[j], cs_ref[j]) for j in range(cs.shape[0]))
    print("  rel err o %.3g final %.3g chunk states %.3g" % (e_o, e_s, e_cs), flush=True)
    assert np.all(np.isfinite(o)) and np.all(np.isfinite(cs)) and np.all(np.isfinite(fs))
    assert e_o <= PARITY_TOL and e_s <= PARITY_TOL and e_cs <= PARITY_TOL
    assert e_o <= SPLIT_TOL and e_s <= SPLIT_TOL and e_cs <= SPLIT_TOL


def test_gdn_zero_length():
    """T = 0: nothing but final_state = state_in (no workspace needed)."""
    H, dk, dv = 2, 128, 32
    inp = gdn_case(7, 0, H, dk, dv)
    S0 = np.random.default_rng(1).standard_normal((H, dk, dv)).astype(np.float32)
    _, _, fs = _run(inp, 0, H, dk, dv, S0=S0)
    assert np.array_equal(fs, S0)


@pytest.mark.parametrize("gv,bv", [(-100.0, None), (0.0, None), (None, 0.0), (None, 1.0), (0.0, 1.0)])
def test_gdn_gate_and_beta_extremes(orc, gv, bv):
    """g = -100 (state wiped every token), g = 0 (no decay), beta = 0 (pure
    decay, nothing written), beta = 1 (full replacement along k_t)."""
    T, H, dk, dv = 130, 2, 128, 32
    inp = gdn_case(11, T, H, dk, dv)
    if gv is not None:
        inp["g"][:] = np.float32(gv)
    if bv is not None:
        inp["beta"][:] = np.float32(bv)
    S0 = np.random.default_rng(5).standard_normal((H, dk, dv)).astype(np.float32)
    o, cs, fs = _run(inp, T, H, dk, dv, S0=S0)
    o_ref, cs_ref, s_ref = _refs(orc, inp, S0=S0)
    e = (rel_err(o, o_ref), rel_err(fs, s_ref), max(rel_err(cs[j], cs_ref[j]) for j in range(cs.shape[0])))
    print("  g %s beta %s: rel err o %.3g final %.3g chunk states %.3g" % ((gv, bv) + e), flush=True)
    assert max(e) <= SPLIT_TOL, (gv, bv, e)


def test_gdn_optional_outputs_and_inplace():
    """chunk_states / final_state may be NULL; final_state may alias
    state_in; none of this changes o by a single bit."""
    import torch
    T, H, dk, dv = 150, 4, 128, 64
    inp = gdn_case(13, T, H, dk, dv)
    S0 = np.random.default_rng(2).standard_normal((H, dk, dv)).astype(np.float32)
    o_a, cs_a, fs_a = _run(inp, T, H, dk, dv, S0=S0)
    o_b, _, _ = _run(inp, T, H, dk, dv, S0=S0, want_cs=False, want_final=False)
    assert np.array_equal(o_a, o_b)
    d = _dev(inp)
    st = torch.from_numpy(S0).cuda()
    o = torch.empty((T, H, dv), dtype=torch.float32, device="cuda")
    cap.gdn_chunked_prefill(d["q"], d["k"], d["v"], d["g"], d["beta"], o, state_in=st, final_state=st)
    torch.cuda.synchronize()
    assert np.array_equal(o.cpu().numpy(), o_a) and np.array_equal(st.cpu().numpy(), fs_a)


def test_gdn_scale():
    T, H, dk, dv = 100, 2, 64, 32
    inp = gdn_case(17, T, H, dk, dv)
    o1, _, _ = _run(inp, T, H, dk, dv, scale=1.0)
    o2, _, _ = _run(inp, T, H, dk, dv, scale=0.125)
    assert np.array_equal(o2, 0.125 * o1)


def test_gdn_deterministic():
    """Two runs give identical bits (no atomics, fixed reduction order)."""
    T, H, dk, dv = 700, 16, 128, 128
    inp = gdn_case(19, T, H, dk, dv)
    a = _run(inp, T, H, dk, dv)
    b = _run(inp, T, H, dk, dv)
    for x, y in zip(a, b):
        assert np.array_equal(x, y)


@pytest.mark.parametrize("split", [64, 128, 192])
def test_gdn_aligned_continuation_is_bitwise(split):
    """A call from the state at an aligned token `split` reproduces the rest of
    one longer call bit for bit: outputs, chunk states and the final state."""
    import torch
    T, H, dk, dv = 320, 4, 128, 64
    inp = gdn_case(23, T, H, dk, dv)
    S0 = np.random.default_rng(3).standard_normal((H, dk, dv)).astype(np.float32)
    o, cs, fs = _run(inp, T, H, dk, dv, S0=S0)
    first = {n: np.ascontiguousarray(inp[n][:split]) for n in ("q", "k", "v", "g", "beta")}
    first.update({n + "_dev": np.ascontiguousarray(inp[n + "_dev"][:split]) for n in ("q", "k", "v")})
    rest = {n: np.ascontiguousarray(inp[n][split:]) for n in ("q", "k", "v", "g", "beta")}
    rest.update({n + "_dev": np.ascontiguousarray(inp[n + "_dev"][split:]) for n in ("q", "k", "v")})
    o1, _, s1 = _run(first, split, H, dk, dv, S0=S0)
    o2, cs2, s2 = _run(rest, T - split, H, dk, dv, S0=s1)
    assert np.array_equal(np.concatenate([o1, o2]), o)
    assert np.array_equal(cs2, cs[split // 64:])
    assert np.array_equal(s2, fs)
    assert torch.cuda.is_available()


def test_gdn_workspace_is_caller_owned(orc):
    """An explicit workspace of exactly gdn_workspace_bytes works, and its
    previous contents do not matter."""
    import torch
    T, H, dk, dv = 190, 2, 64, 32
    inp = gdn_case(29, T, H, dk, dv)
    d = _dev(inp)
    need = cap.gdn_workspace_bytes(T, H)
    assert need == 3 * H * 12800
    ws = torch.full((need,), 0x7F, dtype=torch.uint8, device="cuda")  # NaN patterns
    o = torch.empty((T, H, dv), dtype=torch.float32, device="cuda")
    fs = torch.empty((H, dk, dv), dtype=torch.float32, device="cuda")
    cap.gdn_chunked_prefill(d["q"], d["k"], d["v"], d["g"], d["beta"], o, final_state=fs, workspace=ws)
    torch.cuda.synchronize()
    o_ref, s_ref = orc.gdn_sequential(inp["q"], inp["k"], inp["v"], inp["g"], inp["beta"])
    assert rel_err(o.cpu().numpy(), o_ref) <= SPLIT_TOL and rel_err(fs.cpu().numpy(), s_ref) <= SPLIT_TOL
    with pytest.raises(cap.CapsuleError) as ei:
        cap.gdn_chunked_prefill(d["q"], d["k"], d["v"], d["g"], d["beta"], o, workspace=ws, workspace_bytes=need - 16)
    assert ei.value.status == cap.CAP_E_SIZE


@pytest.mark.parametrize("dk,dv", [(128, 128), (64, 32)])
def test_gdn_one_token_agrees_with_chunked(dk, dv):
    """A one-token prefill from a chunk boundary is the chunked path's
    one-token chunk: token 64 of one 65-token call against a one-token call
    from that call's chunk state 1 -- state and o equal bit for bit, chunk
    state 0 = the entering state.  The decode step (one launch, no workspace)
    agrees to fp32 rounding."""
    import torch
    T, H = 65, 4
    inp = gdn_case(47, T, H, dk, dv)
    S0 = np.random.default_rng(13).standard_normal((H, dk, dv)).astype(np.float32)
    o, cs, fs = _run(inp, T, H, dk, dv, S0=S0)
    d = _dev(inp)
    st = torch.from_numpy(cs[1]).cuda()
    o1 = torch.empty((1, H, dv), dtype=torch.float32, device="cuda")
    cs1 = torch.empty((1, H, dk, dv), dtype=torch.float32, device="cuda")
    fs1 = torch.empty((H, dk, dv), dtype=torch.float32, device="cuda")
    cap.gdn_chunked_prefill(d["q"][64:], d["k"][64:], d["v"][64:], d["g"][64:], d["beta"][64:], o1, state_in=st,
                            chunk_states=cs1, final_state=fs1, T=1, H=H, dk=dk, dv=dv)
    o2 = torch.empty((1, H, dv), dtype=torch.float32, device="cuda")
    fs2 = torch.empty((H, dk, dv), dtype=torch.float32, device="cuda")
    cap.gdn_decode_step(d["q"][64:], d["k"][64:], d["v"][64:], d["g"][64:], d["beta"][64:], o2, state_in=st,
                        final_state=fs2, T=1, H=H, dk=dk, dv=dv)
    torch.cuda.synchronize()
    assert np.array_equal(cs1.cpu().numpy()[0], cs[1])
    assert np.array_equal(fs1.cpu().numpy(), fs)
    assert np.array_equal(o1.cpu().numpy()[0], o[64])
    assert rel_err(fs2.cpu().numpy(), fs) <= SPLIT_TOL
    assert rel_err(o2.cpu().numpy()[0], o[64]) <= SPLIT_TOL


@pytest.mark.parametrize("gv,bv", [(-100.0, None), (None, 0.0), (None, 1.0)])
def test_gdn_one_token_extremes_and_inplace(orc, gv, bv):
    """One-token calls at g = -100 (state wiped), beta = 0 (pure decay) and
    beta = 1 (full replacement along k), updating the state in place."""
    import torch
    H, dk, dv = 3, 128, 64
    inp = gdn_case(53, 1, H, dk, dv)
    if gv is not None:
        inp["g"][:] = np.float32(gv)
    if bv is not None:
        inp["beta"][:] = np.float32(bv)
    S0 = np.random.default_rng(17).standard_normal((H, dk, dv)).astype(np.float32)
    d = _dev(inp)
    st = torch.from_numpy(S0).cuda()
    o = torch.empty((1, H, dv), dtype=torch.float32, device="cuda")
    cap.gdn_chunked_prefill(d["q"], d["k"], d["v"], d["g"], d["beta"], o, state_in=st, final_state=st)
    st2 = torch.from_numpy(S0).cuda()
    o2 = torch.empty((1, H, dv), dtype=torch.float32, device="cuda")
    cap.gdn_decode_step(d["q"], d["k"], d["v"], d["g"], d["beta"], o2, state_in=st2, final_state=st2)
    torch.cuda.synchronize()
    o_ref, s_ref = orc.gdn_sequential(inp["q"], inp["k"], inp["v"], inp["g"], inp["beta"], S0=S0)
    e = (rel_err(o.cpu().numpy(), o_ref), rel_err(st.cpu().numpy(), s_ref),
         rel_err(o2.cpu().numpy(), o_ref), rel_err(st2.cpu().numpy(), s_ref))
    print("  g %s beta %s: rel err o %.3g state %.3g (decode step: o %.3g state %.3g)" % ((gv, bv) + e), flush=True)
    assert max(e) <= SPLIT_TOL, e
