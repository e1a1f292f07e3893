"""Append and the decode path as one graph (GPU, through the C ABI).

cap_set_append against the oracle, bit for bit (positional rows, sliding
windows, untouched buffers, overflow); then §3 Algorithm 1's restore path --
copy the capsule back, append the suffix -- recorded as ONE HIP graph for
the hybrid8 workload (restore + 32 decode steps, each an append of the
token's K/V rows and conv inputs plus six one-token scans) and replayed:
every replay equals the eager cold path bit for bit, with eager work and
synchronisations between the replays; and the same with an unaligned
boundary, where the graph also re-prefills the remainder past P' (both
mixers)."""
import numpy as np
import pytest

import paper_2606_20537_amd as cap
import synth
from gpu_util import device_bytes
from harness import HybridStack, make_inputs

pytestmark = pytest.mark.gpu

# positional rows of 2 KiB and 20 KiB (wider than a copy tile), windows of
# 4 x 8 KiB and 3 x 48 B, and a fixed state the append never touches
LAYOUT = [
    ("kv.k", 2048, 300, cap.CAP_KIND_POSITIONAL),
    ("conv0", 8192, 4, cap.CAP_KIND_FIXED),
    ("state", 4096, 1, cap.CAP_KIND_FIXED),
    ("kv.v", 20480, 64, cap.CAP_KIND_POSITIONAL),
    ("conv1", 48, 3, cap.CAP_KIND_FIXED),
]
SOURCE = [True, True, False, True, True]


def _code(fn, *a):
    try:
        fn(*a)
    except cap.CapsuleError as e:
        return e.status
    return cap.CAP_OK


def test_append_matches_oracle(orc):
    import torch
    bufs = [(n, device_bytes(rb * rows, seed=40 + i, name=n), rb, rows, k) for i, (n, rb, rows, k) in enumerate(LAYOUT)]
    live = cap.cap_set_create(bufs, 64, 1)
    host = [b[1].cpu().numpy() for b in bufs]
    rb = [b[2] for b in bufs]
    rt = [b[3] for b in bufs]
    kd = [b[4] for b in bufs]
    pos = 7
    cap.cap_set_set_position(live, pos)
    for step, n in enumerate([1, 3, 4, 9, 1, 30]):
        srcs_h = [np.random.default_rng(100 + step * 7 + i).integers(0, 256, n * rb[i], dtype=np.uint8)
                  if SOURCE[i] else None for i in range(len(LAYOUT))]
        srcs_d = [None if x is None else torch.from_numpy(x).cuda() for x in srcs_h]
        cap.cap_set_append(live, srcs_d, n)
        assert orc.append(host, srcs_h, rb, rt, kd, pos, n) == 0
        pos += n
        assert cap.cap_set_get_position(live) == pos
        torch.cuda.synchronize()
        for b, h in zip(bufs, host):
            assert np.array_equal(b[1].cpu().numpy(), h), (step, n, b[0])
    # the value rows hold 64: 64 - pos more tokens overflow, nothing is written
    n = 64 - pos + 1
    srcs_d = [torch.zeros(n * rb[i], dtype=torch.uint8, device="cuda") if SOURCE[i] else None for i in range(len(LAYOUT))]
    assert _code(cap.cap_set_append, live, srcs_d, n) == cap.CAP_E_SIZE
    bad = [x for x in srcs_d]
    bad[0] = bufs[2][1]  # a source inside a live buffer
    assert _code(cap.cap_set_append, live, bad, 1) == cap.CAP_E_INVAL
    torch.cuda.synchronize()
    for b, h in zip(bufs, host):
        assert np.array_equal(b[1].cpu().numpy(), h), b[0]
    assert cap.cap_set_get_position(live) == pos


def _snapshot_of(st):
    return ([o.clone() for o in st.o], [s.clone() for s in st.state], [c.clone() for c in st.conv],
            [k.clone() for k in st.kv])


def test_restore_then_decode_as_one_graph():
    import torch
    w = synth.get_config("hybrid8")
    P, n_steps = 2048, w.continuation
    F = P + n_steps
    inputs = make_inputs(w, F, w.seed)
    # eager reference: cold prefill of P tokens, then 32 decode steps
    cold = HybridStack(w, F, inputs=inputs)
    cold.prefill(0, P)
    cold.decode(n_steps)
    torch.cuda.synchronize()
    ref = _snapshot_of(cold)
    # the session whose capsule is restored
    warm = HybridStack(w, F, inputs=inputs)
    warm.prefill(0, P)
    d = cap.capsule_digest_tokens(synth.token_ids(w.seed, P))
    c = warm.snapshot(P, d)
    torch.cuda.synchronize()
    # record restore + 32 decode steps as one graph on a side stream
    g = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        with torch.cuda.graph(g, stream=side):
            warm.restore(c, d)
            warm.decode(n_steps)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    for replay in range(3):
        warm.poison()                          # eager work between replays
        junk = torch.randn(1 << 20, device="cuda").sum()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = _snapshot_of(warm)
        for l, (a, b) in enumerate(zip(got[0], ref[0])):
            assert torch.equal(a[P:F], b[P:F]), (replay, "o", l)
        for kind, xs, ys in (("state", got[1], ref[1]), ("conv", got[2], ref[2])):
            for l, (a, b) in enumerate(zip(xs, ys)):
                assert torch.equal(a, b), (replay, kind, l)
        for l, (a, b) in enumerate(zip(got[3], ref[3])):
            assert torch.equal(a[:F], b[:F]), (replay, "kv", l)
        assert bool(torch.isfinite(junk))


@pytest.mark.parametrize("mixer", ["linattn", "gdn"])
def test_restore_remainder_prefill_and_decode_as_one_graph(mixer):
    """A boundary that is not chunk-aligned (P = 2111, P' = 2048): restore,
    the chunked prefill of the remainder [P', P) in every linear layer with
    its append, then 32 decode steps, recorded as ONE graph (§3 Algorithm 1:
    restore, then re-prefill the tokens past the boundary and append) and
    replayed with eager work between replays; every replay equals the eager
    cold prefill of [0, P) plus the same decode steps, bit for bit (§5: the
    restored state sits on a chunk boundary)."""
    import torch
    w = synth.get_config("hybrid8")
    P, n_steps = 2111, w.continuation
    Pa = (P // w.chunk) * w.chunk
    F = P + n_steps
    inputs = make_inputs(w, F, w.seed, mixer)
    cold = HybridStack(w, F, inputs=inputs, mixer=mixer)
    cold.prefill(0, P)
    cold.decode(n_steps)
    torch.cuda.synchronize()
    ref = _snapshot_of(cold)
    warm = HybridStack(w, F, inputs=inputs, mixer=mixer)
    warm.prefill(0, Pa)
    d = cap.capsule_digest_tokens(synth.token_ids(w.seed, P))
    c = warm.snapshot(P, d)
    warm.prefill(Pa, P)                        # the session went on past the boundary
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        with torch.cuda.graph(g, stream=side):
            assert warm.restore(c, d) == Pa
            warm.prefill(Pa, P)
            warm.decode(n_steps)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    for replay in range(3):
        warm.poison()
        junk = torch.randn(1 << 20, device="cuda").sum()
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = _snapshot_of(warm)
        for l, (a, b) in enumerate(zip(got[0], ref[0])):
            assert torch.equal(a[Pa:F], b[Pa:F]), (replay, "o", l)
        for kind, xs, ys in (("state", got[1], ref[1]), ("conv", got[2], ref[2])):
            for l, (a, b) in enumerate(zip(xs, ys)):
                assert torch.equal(a, b), (replay, kind, l)
        for l, (a, b) in enumerate(zip(got[3], ref[3])):
            assert torch.equal(a[:F], b[:F]), (replay, "kv", l)
        assert bool(torch.isfinite(junk))
