"""Capsules over a Gated-DeltaNet hybrid stack (GPU, through the C ABI).

The paper's model keeps Gated DeltaNet states in its linear layers (§2, §7);
its capsule freezes them together with the KV prefixes and conv tails at a
chunk-aligned boundary (§3 Algorithm 1, §5).  With the hybrid8 shapes and the
delta-rule prefill in every linear layer: restore then continue equals a cold
prefill bit for bit -- outputs, states, conv tails and K/V -- for an aligned
boundary and for one that snapshot floors to the chunk grid, after the live
set has been overwritten; decode steps after the restore match too; and the
cold path matches the oracle's recurrence on sampled heads."""
import numpy as np
import pytest
import torch

import paper_2606_20537_amd as cap
import synth
from gpu_util import PARITY_TOL, rel_err
from harness import HybridStack, make_inputs

pytestmark = pytest.mark.gpu

HYB8 = synth.get_config("hybrid8")


def digest_of(w, P):
    return cap.capsule_digest_tokens(synth.token_ids(w.seed, P))


def assert_same(a, b, t0, t1):
    for l in range(len(a.o)):
        assert torch.equal(a.o[l][t0:t1], b.o[l][t0:t1]), "layer %d outputs differ" % l
    for x, y in zip(a.state, b.state):
        assert torch.equal(x, y)
    for x, y in zip(a.conv, b.conv):
        assert torch.equal(x, y)
    for x, y in zip(a.kv, b.kv):
        assert torch.equal(x[:t1], y[:t1])


@pytest.fixture(scope="module")
def inputs_gdn():
    return make_inputs(HYB8, 2048 + 128 + 8, HYB8.seed + 7, mixer="gdn")


@pytest.mark.parametrize("P", [2048, 2111])
def test_gdn_stack_restore_then_continue_equals_cold(orc, inputs_gdn, P):
    w = HYB8
    Pa = (P // w.chunk) * w.chunk
    F = 2048 + 128
    print("P", P, "aligned", Pa, flush=True)
    cold = HybridStack(w, F + 8, inputs=inputs_gdn, mixer="gdn")
    cold.prefill(0, F)
    cold.decode(8)
    warm = HybridStack(w, F + 8, inputs=inputs_gdn, mixer="gdn")
    warm.prefill(0, Pa)
    # a capsule asked for at P holds the state at P' (the set sits there)
    c = warm.snapshot(P, digest_of(w, P))
    warm.prefill(Pa, F)         # the session goes on past P ...
    warm.poison()               # ... and its live set is overwritten
    assert warm.restore(c, digest_of(w, P)) == Pa
    warm.prefill(Pa, F)
    warm.decode(8)
    torch.cuda.synchronize()
    assert_same(cold, warm, Pa, F + 8)
    # the cold path itself against the oracle's recurrence on two heads of layer 0
    h = cold.inp["lin"][0]["host"]
    heads = [0, 9]
    sub = {n: np.ascontiguousarray(h[n][: F + 8][:, heads]) for n in ("q", "k", "v", "g", "beta")}
    o_ref, s_ref = orc.gdn_sequential(sub["q"], sub["k"], sub["v"], sub["g"], sub["beta"])
    assert rel_err(cold.o[0][:, heads].cpu().numpy(), o_ref) <= PARITY_TOL
    assert rel_err(cold.state[0][heads].cpu().numpy(), s_ref) <= PARITY_TOL
