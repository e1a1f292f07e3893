"""Full-size cases in the launch configuration bench.py times: one 48-layer
workload layer (16384 tokens x 32 heads, dk = dv = 128) of the
linear-attention scan and of the gated delta-rule scan against the oracle on
sampled heads, the full 881,983,488-byte capsule against the oracle's memcpy,
fork x4, and the robot-reset workload (32 environments, gallery of 8
capsules, 1000 batched gather-restores)."""
import numpy as np
import pytest
import torch

import paper_2606_20537_amd as cap
import synth
from gpu_util import PARITY_TOL, SPLIT_TOL, by_head, dev_inputs, elem_err, rel_err

pytestmark = pytest.mark.gpu

H48 = synth.get_config("hybrid48")


def _compare_all_heads(o, cs, fs, per_head_ref, H):
    """Normwise max relative error of o, the final state and every chunk
    state over all heads, from per-head oracle results (o, chunk states,
    final); also the elementwise error (floor 1e-3 of the tensor's scale) of
    o, reported.  Heads are compared one at a time to bound host memory."""
    num = {"o": 0.0, "s": 0.0, "c": 0.0}
    den = {"o": 0.0, "s": 0.0, "c": 0.0}
    elem_o = 0.0
    for h in range(H):
        o_ref, cs_ref, s_ref = per_head_ref[h]
        pairs = {"o": (o[:, h].cpu().numpy(), o_ref[:, 0]), "s": (fs[h].cpu().numpy(), s_ref[0]),
                 "c": (cs[:, h].cpu().numpy(), cs_ref[:, 0])}
        for key, (x, y) in pairs.items():
            num[key] = max(num[key], float(np.max(np.abs(x.astype(np.float64) - y))))
            den[key] = max(den[key], float(np.max(np.abs(y))))
        elem_o = max(elem_o, elem_err(pairs["o"][0], pairs["o"][1]))
    return {k: num[k] / den[k] for k in num}, elem_o


def test_hybrid48_layer_all_heads(orc):
    """One 48-layer-workload layer (16384 tokens x 32 heads, dk = dv = 128) in
    the launch configuration bench.py times: o, the final state and all 256
    chunk states of every head against the oracle (chunked form, itself
    pinned to the recurrence; heads run in parallel threads)."""
    w = H48
    T, H, dk, dv = w.prefix, w.heads, w.dk, w.dv
    inp = synth.linattn_inputs(w.seed, 0, T, H, dk, dv, "bf16")
    d = dev_inputs(inp)
    n_chunks = T // 64
    o = torch.empty((T, H, dv), dtype=torch.float32, device="cuda")
    cs = torch.empty((n_chunks, H, dk, dv), dtype=torch.float32, device="cuda")
    fs = torch.empty((H, dk, dv), dtype=torch.float32, device="cuda")
    cap.linattn_chunked_prefill(d["q"], d["k"], d["v"], d["g"], o, chunk_states=cs, final_state=fs)
    torch.cuda.synchronize()
    assert torch.isfinite(o).all() and torch.isfinite(cs).all()
    ref = by_head(lambda q, k, v, g: orc.chunked(q, k, v, g, 64), [inp[n] for n in ("q", "k", "v", "g")], range(H))
    e, e_elem = _compare_all_heads(o, cs, fs, ref, H)
    print("16k x 32 heads, all heads: rel err o %.3g final %.3g chunk states %.3g; elementwise o %.3g"
          % (e["o"], e["s"], e["c"], e_elem))
    assert max(e.values()) <= PARITY_TOL
    assert max(e.values()) <= SPLIT_TOL
    # the final-state-only call (the cold-prefill configuration bench.py
    # times for TTFT) takes its own instantiation: same o and final state
    o2 = torch.empty_like(o)
    fs2 = torch.empty_like(fs)
    cap.linattn_chunked_prefill(d["q"], d["k"], d["v"], d["g"], o2, final_state=fs2)
    torch.cuda.synchronize()
    assert torch.equal(o2, o) and torch.equal(fs2, fs)


def test_hybrid48_gdn_layer_all_heads(orc):
    """The delta-rule prefill at the same layer shape, one call over all 16384
    tokens: o, all 256 chunk states and the final state of every head against
    the oracle's chunked (WY) form, itself pinned to the token-by-token
    recurrence."""
    w = H48
    T, H, dk, dv = w.prefix, w.heads, w.dk, w.dv
    inp = synth.gdn_inputs(w.seed, 0, T, H, dk, dv, "bf16")
    d = dev_inputs(inp)
    beta = torch.from_numpy(inp["beta"]).cuda()
    n_chunks = T // 64
    o = torch.empty((T, H, dv), dtype=torch.float32, device="cuda")
    cs = torch.empty((n_chunks, H, dk, dv), dtype=torch.float32, device="cuda")
    fs = torch.empty((H, dk, dv), dtype=torch.float32, device="cuda")
    cap.gdn_chunked_prefill(d["q"], d["k"], d["v"], d["g"], beta, o, chunk_states=cs, final_state=fs)
    torch.cuda.synchronize()
    assert torch.isfinite(o).all() and torch.isfinite(cs).all()
    ref = by_head(lambda q, k, v, g, b: orc.gdn_chunked(q, k, v, g, b, 64),
                  [inp[n] for n in ("q", "k", "v", "g", "beta")], range(H))
    e, e_elem = _compare_all_heads(o, cs, fs, ref, H)
    print("gdn 16k x 32 heads, all heads: rel err o %.3g final %.3g chunk states %.3g; elementwise o %.3g"
          % (e["o"], e["s"], e["c"], e_elem))
    assert max(e.values()) <= PARITY_TOL
    assert max(e.values()) <= SPLIT_TOL


def hybrid48_layout(w):
    """(name, row_bytes, rows, kind) of the 48-layer live set, 3:1 interleaved."""
    lay = []
    li = ki = 0
    for layer in range(w.n_linear + w.n_full):
        if layer % 4 == 3:
            for n in ("k", "v"):
                lay.append(("kv%d.%s" % (ki, n), w.kv_row_bytes, w.t_max, cap.CAP_KIND_POSITIONAL))
            ki += 1
        else:
            lay.append(("lin%d.state" % li, w.heads * w.dk * w.dv * 4, 1, cap.CAP_KIND_FIXED))
            lay.append(("lin%d.conv" % li, w.conv_width * w.conv_channels * 2, 1, cap.CAP_KIND_FIXED))
            li += 1
    return lay


def random_buffers(layout, seed):
    g = torch.Generator(device="cuda").manual_seed(seed)
    out = []
    for name, rb, rows, kind in layout:
        t = torch.empty(rb * rows, dtype=torch.uint8, device="cuda")
        t.view(torch.int32).random_(generator=g)
        out.append((name, t, rb, rows, kind))
    return out


def test_hybrid48_capsule_bytes_restore_and_fork(orc):
    w = H48
    P = w.prefix
    layout = hybrid48_layout(w)
    bufs = random_buffers(layout, 1)
    live = cap.cap_set_create(bufs, w.chunk, 7)
    cap.cap_set_set_position(live, P)
    nbytes = cap.capsule_bytes(live, P)
    assert nbytes == 881_983_488
    arena = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    c = cap.capsule_snapshot(live, P, 1, arena)
    torch.cuda.synchronize()
    host = [b[1].cpu().numpy() for b in bufs]
    rb, rt, kd = [b[2] for b in bufs], [b[3] for b in bufs], [b[4] for b in bufs]
    want = orc.snapshot(host, rb, rt, kd, P)
    assert np.array_equal(arena.cpu().numpy(), want)
    # dirty everything, restore, compare with the oracle's restore of the same bytes
    for b in bufs:
        b[1].fill_(0xA5)
    cap.capsule_restore(c, live, 1)
    torch.cuda.synchronize()
    expect = [np.full_like(h, 0xA5) for h in host]
    orc.restore(want, expect, rb, rt, kd, P)
    for b, e in zip(bufs, expect):
        assert np.array_equal(b[1].cpu().numpy(), e), b[0]
    # fork into 4 sibling sessions
    sibs = []
    for i in range(4):
        sb = random_buffers(layout, 10 + i)
        sibs.append((cap.cap_set_create(sb, w.chunk, 7), sb))
    cap.capsule_fork(c, [s for s, _ in sibs], 1)
    torch.cuda.synchronize()
    for s, sb in sibs:
        for (name, t, r, rows, kind), src in zip(sb, bufs):
            n = P * r if kind == cap.CAP_KIND_POSITIONAL else r * rows
            assert torch.equal(t[:n], src[1][:n]), name


def _bf16_dev(bits):
    return torch.from_numpy(bits.view(np.int16).copy()).view(torch.bfloat16).cuda()


def test_hybrid48_fork_branches_continue_like_cold():
    """Fork of the 16384-token 48-layer capsule into 4 sessions, each
    continuing with its own 64-token suffix (§3 "Four verbs" (iii)): every
    branch equals, bit for bit, the cold prefill of its own 16448 tokens (o of
    the suffix and the final state of all 36 linear layers, the K/V rows of
    the 24 positional buffers and the 36 conv windows), and the branches
    differ from each other.  Layer l reads the inputs of distinct layer l % 4
    (4 distinct layers, as in bench.py)."""
    w = H48
    P, n_sfx, nd, n_br = w.prefix, 64, 4, 4
    F = P + n_sfx
    H, dk, dv = w.heads, w.dk, w.dv
    W, Cc = w.conv_width, w.conv_channels
    # base inputs of the 4 distinct layers over [0, F), and per branch the
    # suffix rows [P, F) from another stream
    base = []
    for l in range(nd):
        inp = synth.linattn_inputs(w.seed, l, F, H, dk, dv, "bf16")
        e = {n: _bf16_dev(inp[n + "_dev"]) for n in ("q", "k", "v")}
        e["g"] = torch.from_numpy(inp["g"]).cuda()
        base.append(e)
        del inp
    sfx = []
    for b in range(n_br):
        per = []
        for l in range(nd):
            inp = synth.linattn_inputs(w.seed + 777 * (b + 1), l, n_sfx, H, dk, dv, "bf16")
            e = {n: _bf16_dev(inp[n + "_dev"]) for n in ("q", "k", "v")}
            e["g"] = torch.from_numpy(inp["g"]).cuda()
            per.append(e)
        sfx.append(per)
    gen = torch.Generator(device="cuda").manual_seed(4848)

    def randn_bf16(*shape):
        return torch.randn(*shape, generator=gen, device="cuda", dtype=torch.float32).to(torch.bfloat16)

    kv_rows = [randn_bf16(w.t_max, w.kv_heads, w.kv_dim) for _ in range(2 * w.n_full)]   # rows [0, P) used
    conv_src = [randn_bf16(W, Cc) for _ in range(w.n_linear)]                           # the tail at P
    kv_sfx = [[randn_bf16(n_sfx, w.kv_heads, w.kv_dim) for _ in range(2 * w.n_full)] for _ in range(n_br)]
    conv_sfx = [[randn_bf16(n_sfx, Cc) for _ in range(w.n_linear)] for _ in range(n_br)]

    def make_set(fill):
        states = [torch.full((H, dk, dv), fill, dtype=torch.float32, device="cuda") for _ in range(w.n_linear)]
        convs = [torch.full((W, Cc), fill, dtype=torch.bfloat16, device="cuda") for _ in range(w.n_linear)]
        kvs = [torch.full((w.t_max, w.kv_heads, w.kv_dim), fill, dtype=torch.bfloat16, device="cuda")
               for _ in range(2 * w.n_full)]
        bufs, li, ki = [], 0, 0
        for layer in range(w.n_linear + w.n_full):
            if layer % 4 == 3:
                for _ in range(2):
                    bufs.append(("kv%d" % ki, kvs[ki], w.kv_row_bytes, w.t_max, cap.CAP_KIND_POSITIONAL))
                    ki += 1
            else:
                bufs.append(("state%d" % li, states[li], H * dk * dv * 4, 1, cap.CAP_KIND_FIXED))
                bufs.append(("conv%d" % li, convs[li], Cc * 2, W, cap.CAP_KIND_FIXED))
                li += 1
        return cap.cap_set_create(bufs, w.chunk, 48), states, convs, kvs, bufs

    # the source session: prefill [0, P) of all 36 layers, K/V rows and conv tail at P
    src, s_states, s_convs, s_kvs, _ = make_set(0.0)
    o_tmp = torch.empty((F, H, dv), dtype=torch.float32, device="cuda")
    for l in range(w.n_linear):
        e = base[l % nd]
        cap.linattn_chunked_prefill(e["q"][:P], e["k"][:P], e["v"][:P], e["g"][:P], o_tmp[:P],
                                    final_state=s_states[l])
        s_convs[l].copy_(conv_src[l])
    for i in range(2 * w.n_full):
        s_kvs[i][:P].copy_(kv_rows[i][:P])
    cap.cap_set_set_position(src, P)
    arena = torch.empty(cap.capsule_bytes(src, P), dtype=torch.uint8, device="cuda")
    c = cap.capsule_snapshot(src, P, 9, arena)
    # fork into 4 poisoned sessions, each continuing [P, F) on its own suffix
    branches = [make_set(float("nan")) for _ in range(n_br)]
    cap.capsule_fork(c, [b[0] for b in branches], 9)
    o_br = []
    for b, (bset, states, convs, kvs, bufs) in enumerate(branches):
        outs = []
        for l in range(w.n_linear):
            e = sfx[b][l % nd]
            ob = torch.empty((n_sfx, H, dv), dtype=torch.float32, device="cuda")
            cap.linattn_chunked_prefill(e["q"], e["k"], e["v"], e["g"], ob, state_in=states[l],
                                        final_state=states[l])
            outs.append(ob)
        srcs, li, ki = [], 0, 0
        for name, *_ in bufs:
            if name.startswith("kv"):
                srcs.append(kv_sfx[b][ki]); ki += 1
            elif name.startswith("conv"):
                srcs.append(conv_sfx[b][li]); li += 1
            else:
                srcs.append(None)
        cap.cap_set_append(bset, srcs, n_sfx)
        o_br.append(outs)
    torch.cuda.synchronize()
    # each branch against its own cold path: one prefill of [0, F) per layer
    work = [{n: t.clone() for n, t in base[l].items()} for l in range(nd)]
    for b, (bset, states, convs, kvs, bufs) in enumerate(branches):
        for l in range(nd):
            for n in ("q", "k", "v", "g"):
                work[l][n][P:F].copy_(sfx[b][l][n])
        cold_state = torch.empty((H, dk, dv), dtype=torch.float32, device="cuda")
        for l in range(w.n_linear):
            e = work[l % nd]
            cap.linattn_chunked_prefill(e["q"], e["k"], e["v"], e["g"], o_tmp, final_state=cold_state)
            torch.cuda.synchronize()
            assert torch.equal(o_br[b][l], o_tmp[P:F]), (b, l)
            assert torch.equal(states[l], cold_state), (b, l)
            # conv window: the last W rows of (tail at P, then the suffix's conv inputs)
            assert torch.equal(convs[l], torch.cat([conv_src[l], conv_sfx[b][l]])[-W:]), (b, l)
        for i in range(2 * w.n_full):
            assert torch.equal(kvs[i][:P], kv_rows[i][:P]), (b, i)
            assert torch.equal(kvs[i][P:F], kv_sfx[b][i]), (b, i)
        assert cap.cap_set_get_position(bset) == F
    assert not torch.equal(o_br[0][0], o_br[1][0])   # distinct suffixes give distinct branches
    print("fork x4 at 16384 tokens, 64-token suffixes: every branch bitwise equal to its cold path")


def test_robot_reset_1000_gather_restores():
    w = synth.get_config("robot_reset")
    ex = dict(w.extra)
    n_env, n_gal, n_resets = ex["envs"], ex["gallery"], ex["resets"]
    layout = []
    for l in range(w.n_full):
        for n in ("k", "v"):
            layout.append(("kv%d.%s" % (l, n), w.kv_row_bytes, w.t_max, cap.CAP_KIND_POSITIONAL))
    layout.append(("denoiser", ex["denoiser_bytes"], 1, cap.CAP_KIND_FIXED))
    P = w.prefix
    gal_bufs, gallery = [], []
    for gi in range(n_gal):
        b = random_buffers(layout, 100 + gi)
        s = cap.cap_set_create(b, w.chunk, 3)
        cap.cap_set_set_position(s, P)
        arena = torch.empty(cap.capsule_bytes(s, P), dtype=torch.uint8, device="cuda")
        gallery.append(cap.capsule_snapshot(s, P, 0, arena))
        gal_bufs.append((s, b))
    assert cap.capsule_info(gallery[0])["bytes"] == 17_137_664
    envs = []
    for e in range(n_env):
        b = random_buffers(layout, 500 + e)
        envs.append((cap.cap_set_create(b, w.chunk, 3), b))
    ids_all = synth.rng(w.seed, 0, "reset_ids").integers(0, n_gal, size=(n_resets, n_env)).astype(np.int32)
    den_gal = torch.stack([b[-1][1] for _, b in gal_bufs])          # [gallery, 2 MiB]
    mismatches = torch.zeros((), dtype=torch.int64, device="cuda")
    for r in range(n_resets):
        ids = ids_all[r]
        cap.capsule_gather_restore(gallery, ids, [s for s, _ in envs])
        den_env = torch.stack([b[-1][1] for _, b in envs])          # [env, 2 MiB]
        mismatches += (den_env != den_gal[torch.from_numpy(ids).long().cuda()]).sum()
        if r % 100 == 99 or r == n_resets - 1:
            for (s, b), i in zip(envs, ids):
                for (name, t, rb, rows, kind), src in zip(b, gal_bufs[i][1]):
                    assert torch.equal(t, src[1]), (r, name)
    assert int(mismatches) == 0


def test_long_sequence_131072_tokens(orc):
    """131,072 tokens in one call (2048 chunks; chunk-state offsets past
    4 GiB, 64-bit chunk bases): o and the final state against the oracle's
    recurrence on every head, and the chunk state entering the last chunk
    equal, bit for bit, to the final state of a call over the first 2047
    chunks."""
    T, H, dk, dv = 131072, 2, 128, 128
    inp = synth.linattn_inputs(H48.seed + 3, 0, T, H, dk, dv, "bf16")
    d = dev_inputs(inp)
    n_chunks = T // 64
    o = torch.empty((T, H, dv), dtype=torch.float32, device="cuda")
    cs = torch.empty((n_chunks, H, dk, dv), dtype=torch.float32, device="cuda")
    fs = torch.empty((H, dk, dv), dtype=torch.float32, device="cuda")
    print("one call over %d tokens" % T, flush=True)
    cap.linattn_chunked_prefill(d["q"], d["k"], d["v"], d["g"], o, chunk_states=cs, final_state=fs)
    Tp = T - 64
    o_p = torch.empty((Tp, H, dv), dtype=torch.float32, device="cuda")
    fs_p = torch.empty((H, dk, dv), dtype=torch.float32, device="cuda")
    cap.linattn_chunked_prefill(d["q"][:Tp], d["k"][:Tp], d["v"][:Tp], d["g"][:Tp], o_p, final_state=fs_p,
                                T=Tp, H=H, dk=dk, dv=dv, in_dtype=cap.CAP_DTYPE_BF16)
    torch.cuda.synchronize()
    assert torch.equal(cs[n_chunks - 1], fs_p)
    assert torch.equal(o[:Tp], o_p)
    print("oracle recurrence over %d tokens x %d heads" % (T, H), flush=True)
    o_ref, s_ref = orc.sequential(inp["q"], inp["k"], inp["v"], inp["g"])
    e_o, e_s = rel_err(o.cpu().numpy(), o_ref), rel_err(fs.cpu().numpy(), s_ref)
    print("rel err o %.3g final %.3g" % (e_o, e_s), flush=True)
    assert e_o <= SPLIT_TOL and e_s <= SPLIT_TOL


def test_capsule_larger_than_4gib():
    """A 5.4 GB capsule (one positional buffer of 1,048,576 valid rows of
    5120 B, then a fixed 2 MiB buffer whose capsule offset lies past 4 GiB):
    snapshot and restore are byte-exact."""
    rb, rows, P = 5120, (1 << 20) + 64, 1 << 20
    big = torch.empty(rb * rows, dtype=torch.uint8, device="cuda")
    big.view(torch.int32).random_(generator=torch.Generator(device="cuda").manual_seed(5))
    st = torch.empty(2 << 20, dtype=torch.uint8, device="cuda")
    st.view(torch.int32).random_(generator=torch.Generator(device="cuda").manual_seed(6))
    bufs = [("kv", big, rb, rows, cap.CAP_KIND_POSITIONAL), ("state", st, 2 << 20, 1, cap.CAP_KIND_FIXED)]
    s = cap.cap_set_create(bufs, 64, 9)
    cap.cap_set_set_position(s, P)
    nbytes = cap.capsule_bytes(s, P)
    assert nbytes == rb * P + (2 << 20) and nbytes > (4 << 30)
    arena = torch.empty(nbytes, dtype=torch.uint8, device="cuda")
    c = cap.capsule_snapshot(s, P, 3, arena)
    torch.cuda.synchronize()
    assert torch.equal(arena[: rb * P], big[: rb * P])
    assert torch.equal(arena[rb * P:], st)
    want_tail = big[rb * P:].clone()
    big.fill_(0xA5)
    st.fill_(0x5A)
    cap.capsule_restore(c, s, 3)
    torch.cuda.synchronize()
    assert torch.equal(big[: rb * P], arena[: rb * P])
    assert torch.equal(st, arena[rb * P:])
    assert bool((big[rb * P:] == 0xA5).all())  # rows past P' are left alone
    del want_tail
