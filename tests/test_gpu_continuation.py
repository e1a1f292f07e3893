"""End-to-end restore / continue on the workload shapes (GPU, through the
C ABI): restore at a chunk-aligned boundary then continue is bit-identical to
a cold prefill (§5), survives a fully dirtied live set (§5), fork branches
and rollback match their cold paths (§3 "Four verbs"), and restoring the KV
alone without the recurrent fold does not (the KV-only ablation of §7.2)."""
import numpy as np
import pytest
import torch

import synth
from gpu_util import PARITY_TOL, by_head, rel_err
from harness import HybridStack, make_inputs

pytestmark = pytest.mark.gpu

HYB8 = synth.get_config("hybrid8")
ALIGN = synth.get_config("align_stress")


def digest_of(w, P):
    import paper_2606_20537_amd as cap
    return cap.capsule_digest_tokens(synth.token_ids(w.seed, P))


def assert_same_outputs(a, b, t0, t1):
    for l in range(len(a.o)):
        assert torch.equal(a.o[l][t0:t1], b.o[l][t0:t1]), "layer %d outputs differ" % l
    for x, y in zip(a.state, b.state):
        assert torch.equal(x, y)
    for x, y in zip(a.conv, b.conv):
        assert torch.equal(x, y)
    for x, y in zip(a.kv, b.kv):
        assert torch.equal(x[:t1], y[:t1])


def test_tiny_restore_then_continue_equals_cold(orc):
    w = synth.get_config("tiny")
    F, P = 256, w.prefix
    cold = HybridStack(w, F)
    cold.prefill(0, F)
    warm = HybridStack(w, F, inputs=cold.inp)
    warm.prefill(0, P)
    c = warm.snapshot(P, digest_of(w, P))
    warm.poison()
    assert warm.restore(c, digest_of(w, P)) == P
    warm.prefill(P, F)
    torch.cuda.synchronize()
    assert_same_outputs(cold, warm, P, F)
    h = cold.inp["lin"][0]["host"]
    o_ref, s_ref = orc.sequential(h["q"], h["k"], h["v"], h["g"])
    assert rel_err(cold.o[0].cpu().numpy(), o_ref) <= PARITY_TOL
    assert rel_err(cold.state[0].cpu().numpy(), s_ref) <= PARITY_TOL


@pytest.fixture(scope="module")
def inputs_hyb8():
    return make_inputs(HYB8, 2048 + 64 + 32, HYB8.seed)


def test_hybrid8_capsule_then_decode_steps(orc, inputs_hyb8):
    """Capsule at 2048, then 32 single-token continuation steps."""
    w, P, n = HYB8, 2048, HYB8.continuation
    F = P + n
    cold = HybridStack(w, F, inputs=inputs_hyb8)
    cold.prefill(0, P)
    cold.decode(n)
    warm = HybridStack(w, F, inputs=inputs_hyb8)
    warm.prefill(0, P)
    d = digest_of(w, P)
    c = warm.snapshot(P, d)
    warm.poison()
    warm.restore(c, d)
    warm.decode(n)
    torch.cuda.synchronize()
    assert_same_outputs(cold, warm, P, F)
    # every layer of the cold path against the oracle (all 2080 tokens)
    for l in range(w.n_linear):
        hh = inputs_hyb8["lin"][l]["host"]
        o_ref, s_ref = orc.sequential(hh["q"][:F], hh["k"][:F], hh["v"][:F], hh["g"][:F])
        assert rel_err(cold.o[l].cpu().numpy(), o_ref) <= PARITY_TOL, l
        assert rel_err(cold.state[l].cpu().numpy(), s_ref) <= PARITY_TOL, l


ALIGN_T = 8192 + 63 + 32
ALIGN_PREFIXES = list(range(1024, 8193, 1024))


@pytest.fixture(scope="module")
def inputs_align():
    return make_inputs(ALIGN, ALIGN_T, ALIGN.seed)


@pytest.fixture(scope="module")
def oracle_align(orc, inputs_align):
    """The oracle's chunked form over every token the sweep uses, per layer
    and head: o for all tokens, and the states entering the chunks at L and
    L + 64 for every swept L (the sweep's final states lie in those chunks)."""
    keep = sorted({L // 64 for L in ALIGN_PREFIXES} | {L // 64 + 1 for L in ALIGN_PREFIXES})
    out = []
    for l in range(ALIGN.n_linear):
        h = inputs_align["lin"][l]["host"]
        arrs = [h[n][:ALIGN_T] for n in ("q", "k", "v", "g")]
        res = by_head(lambda q, k, v, g: orc.chunked(q, k, v, g, 64), arrs, range(ALIGN.heads))
        o = np.concatenate([r[0] for r in res], axis=1)
        cs = {j: np.concatenate([r[1][j] for r in res], axis=0) for j in keep}
        out.append({"o": o, "cs": cs})
    return out


def oracle_state_at(orc, inputs, ref, l, F):
    """The oracle's state after token F - 1 of layer l: the chunked form's
    state entering the chunk of F, advanced token by token by the sequential
    recurrence."""
    j = F // 64
    h = inputs["lin"][l]["host"]
    sub = [np.ascontiguousarray(h[n][64 * j:F]) for n in ("q", "k", "v", "g")]
    _, S = orc.sequential(*sub, S0=ref[l]["cs"][j])
    return S


@pytest.mark.parametrize("L", ALIGN_PREFIXES)
@pytest.mark.parametrize("off", [0, 2, 63])
def test_alignment_sweep(orc, inputs_align, oracle_align, L, off):
    """Snapshot requested at P = L + off (P' = L): restore then re-prefill the
    remainder [P', P + 32) equals the cold prefill bit for bit; the cold run
    itself matches the oracle (o over [P', P + 32) and every layer's final
    state, max relative error 2e-3)."""
    w = ALIGN
    P = L + off
    F = P + 32
    cold = HybridStack(w, F, inputs=inputs_align)
    cold.prefill(0, F)
    warm = HybridStack(w, F, inputs=inputs_align)
    warm.prefill(0, L)
    d = digest_of(w, P)
    c = warm.snapshot(P, d)
    if off:
        warm.prefill(L, P)  # the session moves on past the boundary
    warm.poison()
    assert warm.restore(c, d) == L
    warm.prefill(L, F)
    torch.cuda.synchronize()
    assert_same_outputs(cold, warm, L, F)
    errs = []
    for l in range(w.n_linear):
        e_o = rel_err(cold.o[l][L:F].cpu().numpy(), oracle_align[l]["o"][L:F])
        e_s = rel_err(cold.state[l].cpu().numpy(), oracle_state_at(orc, inputs_align, oracle_align, l, F))
        errs.append(max(e_o, e_s))
    print("L %d off %d: max rel err vs oracle over 6 layers %.3g" % (L, off, max(errs)))
    assert max(errs) <= PARITY_TOL


@pytest.mark.parametrize("mixer", ["linattn", "gdn"])
def test_one_token_remainder_then_decode(inputs_hyb8, mixer):
    """A snapshot requested one token past a chunk boundary (P = P' + 1):
    restore P', re-prefill the one-token remainder as its own call, then
    decode -- equal bit for bit to a cold session that prefilled [0, P) in
    one call and decoded the same tokens."""
    w = HYB8
    L, n = 2048, 4
    P = L + 1
    F = P + n
    inp = inputs_hyb8 if mixer == "linattn" else make_inputs(w, F, w.seed + 5, mixer)
    cold = HybridStack(w, F, inputs=inp, mixer=mixer)
    cold.prefill(0, P)
    cold.decode(n)
    warm = HybridStack(w, F, inputs=inp, mixer=mixer)
    warm.prefill(0, L)
    d = digest_of(w, P)
    c = warm.snapshot(P, d)
    warm.prefill(L, P)
    warm.poison()
    assert warm.restore(c, d) == L
    warm.prefill(L, P)   # the remainder: one token, one call
    warm.decode(n)
    torch.cuda.synchronize()
    assert_same_outputs(cold, warm, L, F)


def test_unaligned_split_is_only_close(inputs_align):
    """Negative control for the alignment rule: continuing from an unaligned
    position P starts a chunk grid the cold prefill never had; results stay
    within tolerance but are not required to match bit for bit (reported)."""
    w = ALIGN
    P, F = 2050, 2050 + 64
    cold = HybridStack(w, F, inputs=inputs_align)
    cold.prefill(0, F)
    warm = HybridStack(w, F, inputs=inputs_align)
    warm.prefill(0, P)
    warm.prefill(P, F)
    torch.cuda.synchronize()
    same = all(torch.equal(a[P:F], b[P:F]) for a, b in zip(cold.o, warm.o))
    err = max(rel_err(a[P:F].cpu().numpy(), b[P:F].cpu().numpy()) for a, b in zip(warm.o, cold.o))
    print("unaligned continuation at %d: bitwise equal %s, max rel diff %.3g" % (P, same, err))
    assert err <= PARITY_TOL


def branch_inputs(base, w, P, F, stream):
    """Inputs equal to `base` on [0, P) and drawn from another stream on [P, F)."""
    other = make_inputs(w, F, w.seed + 777 * stream)
    out = {"lin": [], "kv": [], "conv": []}
    for a, b in zip(base["lin"], other["lin"]):
        e = {}
        for n in ("q", "k", "v", "g"):
            e[n] = torch.cat([a[n][:P], b[n][P:F]]).contiguous()
        out["lin"].append(e)
    for key in ("kv", "conv"):
        for a, b in zip(base[key], other[key]):
            out[key].append(torch.cat([a[:P], b[P:F]]).contiguous())
    return out


def test_fork_branches_match_their_cold_paths(inputs_hyb8):
    import paper_2606_20537_amd as cap
    w, P, F = HYB8, 2048, 2048 + 64
    src = HybridStack(w, F, inputs=inputs_hyb8)
    src.prefill(0, P)
    d = digest_of(w, P)
    c = src.snapshot(P, d)
    branches = [HybridStack(w, F, inputs=branch_inputs(inputs_hyb8, w, P, F, i + 1)) for i in range(4)]
    for b in branches:
        b.poison()
    cap.capsule_fork(c, [b.set for b in branches], d)
    outs = []
    for i, b in enumerate(branches):
        b.pos = P
        b.prefill(P, F)
        cold = HybridStack(w, F, inputs=b.inp)
        cold.prefill(0, F)
        torch.cuda.synchronize()
        assert_same_outputs(cold, b, P, F)
        outs.append(b.o[0][P:F].clone())
    assert not torch.equal(outs[0], outs[1])  # distinct suffixes give distinct branches


def test_rollback_to_earlier_boundary(inputs_hyb8):
    w, P, F = HYB8, 2048, 2048 + 64
    inp_a = branch_inputs(inputs_hyb8, w, P, F, 11)
    inp_b = branch_inputs(inputs_hyb8, w, P, F, 12)
    st = HybridStack(w, F, inputs=inp_a)
    st.prefill(0, P)
    d = digest_of(w, P)
    c_early = st.snapshot(P, d)
    st.prefill(P, F)                      # descend along A
    c_late = st.snapshot(F, 99)
    st.restore(c_early, d)                # roll back to P
    st.inp = inp_b
    st.prefill(P, F)                      # descend along B
    cold_b = HybridStack(w, F, inputs=inp_b)
    cold_b.prefill(0, F)
    torch.cuda.synchronize()
    assert_same_outputs(cold_b, st, P, F)
    st.restore(c_late, 99)                # and forward again to the end of A
    cold_a = HybridStack(w, F, inputs=inp_a)
    cold_a.prefill(0, F)
    torch.cuda.synchronize()
    for x, y in zip(st.state, cold_a.state):
        assert torch.equal(x, y)


@pytest.mark.parametrize("mode", ["zeroed", "stale"])
def test_kv_only_restore_diverges(inputs_hyb8, mode):
    """Restoring the positional KV without the recurrent fold and conv tails
    (the KV-only ablation) does not reproduce the cold continuation."""
    w, P, F = HYB8, 2048, 2048 + 32
    cold = HybridStack(w, F, inputs=inputs_hyb8)
    cold.prefill(0, F)
    warm = HybridStack(w, F, inputs=inputs_hyb8)
    warm.prefill(0, P)
    c = warm.snapshot(P, 0)
    stale = HybridStack(w, F, inputs=make_inputs(w, P, w.seed + 4242))
    stale.prefill(0, P)
    warm.restore(c, 0)
    for l in range(w.n_linear):
        if mode == "zeroed":
            warm.state[l].zero_()
            warm.conv[l].zero_()
        else:
            warm.state[l].copy_(stale.state[l])
            warm.conv[l].copy_(stale.conv[l])
    warm.prefill(P, F)
    torch.cuda.synchronize()
    for x, y in zip(warm.kv, cold.kv):   # the KV region itself is restored exactly
        assert torch.equal(x[:F], y[:F])
    err = max(rel_err(a[P:F].cpu().numpy(), b[P:F].cpu().numpy()) for a, b in zip(warm.o, cold.o))
    print("KV-only (%s fold): max rel diff of continuation outputs %.3g" % (mode, err))
    assert err > 100 * PARITY_TOL
