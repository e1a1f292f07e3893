"""Pins for the CPU oracle: checks against what the mathematics and the paper
fix, independent of the oracle's own code.

Each pin is a plain function ``pin_*(orc)`` that raises AssertionError on a
violation, so that the same pins run against the default oracle build
(tests/test_oracle_pins.py) and against deliberately broken copies of it
(tests/test_oracle_mutants.py, which shows that plausible mistakes -- a
dropped term, a wrong sign or index, a transposed operand -- are caught).
"""
import os

import numpy as np

from synth import rng

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


# --------------------------------------------------------------- helpers ----
def _inputs(seed, T, H, dk, dv, gate="real"):
    r = rng(seed, 0, "pin")
    q = r.standard_normal((T, H, dk)).astype(np.float32)
    k = r.standard_normal((T, H, dk)).astype(np.float32)
    v = r.standard_normal((T, H, dv)).astype(np.float32)
    if gate == "real":
        x = r.normal(3.0, 0.5, size=(T, H))
        g = (-np.log1p(np.exp(-x))).astype(np.float32)
    elif gate == "wide":
        g = r.uniform(-2.0, 0.0, size=(T, H)).astype(np.float32)
    else:
        g = np.full((T, H), float(gate), np.float32)
    S0 = r.standard_normal((H, dk, dv))
    return q, k, v, g, S0


def _rel(a, b):
    """max |a - b| / max |b| (0 when both are empty or zero)."""
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    if a.size == 0:
        return 0.0
    den = np.max(np.abs(b))
    num = np.max(np.abs(a - b))
    return float(num / den) if den > 0 else float(num)


def _both_forms(orc, q, k, v, g, S0, C, scale=1.0):
    o_s, S_s = orc.sequential(q, k, v, g, S0=S0, scale=scale)
    o_c, _, S_c = orc.chunked(q, k, v, g, C, S0=S0, scale=scale)
    return (o_s, S_s), (o_c, S_c)


# ------------------------------------------------------- scan: closed forms --
def pin_counting_scalar(orc):
    """dk = dv = 1, q = k = v = 1, no decay (g = 0): the state is a running
    count, o_t = s0 + t + 1 exactly (integers are exact in fp64)."""
    for C in (1, 3, 64):
        for T in (1, 5, 130):
            ones = np.ones((T, 1, 1), np.float32)
            g = np.zeros((T, 1), np.float32)
            S0 = np.full((1, 1, 1), 7.0)
            want = 7.0 + np.arange(1, T + 1, dtype=np.float64)
            (o_s, S_s), (o_c, S_c) = _both_forms(orc, ones, ones, ones, g, S0, C)
            assert np.array_equal(o_s[:, 0, 0], want), "sequential counting"
            assert np.array_equal(o_c[:, 0, 0], want), "chunked counting"
            assert S_s[0, 0, 0] == want[-1] and S_c[0, 0, 0] == want[-1]


def pin_halving_scalar(orc):
    """dk = dv = 1, q = k = v = 1, decay a = exp(g) with g = log(1/2) rounded to
    fp32: s_t = sum_{m<=t} a^(t-m) = (1 - a^(t+1)) / (1 - a) (geometric
    series), within fp32's rounding of log(1/2) of the ideal 2 - 2^-t."""
    T = 40
    ones = np.ones((T, 1, 1), np.float32)
    g = np.full((T, 1), np.float32(np.log(0.5)), np.float32)
    a = np.exp(np.float64(g[0, 0]))
    t = np.arange(T, dtype=np.float64)
    closed = (1.0 - a ** (t + 1)) / (1.0 - a)
    ideal = 2.0 - 2.0 ** (-t)
    for C in (1, 4, 64):
        (o_s, _), (o_c, _) = _both_forms(orc, ones, ones, ones, g, None, C)
        assert _rel(o_s[:, 0, 0], closed) < 1e-13
        assert _rel(o_c[:, 0, 0], closed) < 1e-13
        assert np.max(np.abs(o_s[:, 0, 0] - ideal)) < 1e-6


def pin_causal_linear_attention(orc):
    """g = 0 reduces the recurrence to causal (unnormalised) linear attention:
    O = tril(Q K^T) V + Q S0 per head (textbook masked form, numpy matmul)."""
    for (T, H, dk, dv, C) in ((37, 2, 8, 5, 4), (130, 1, 16, 16, 64), (64, 3, 4, 12, 16)):
        q, k, v, g, S0 = _inputs(11 + T, T, H, dk, dv, gate=0.0)
        (o_s, S_s), (o_c, S_c) = _both_forms(orc, q, k, v, g, S0, C)
        for h in range(H):
            Q, K, V = (x[:, h, :].astype(np.float64) for x in (q, k, v))
            want = np.tril(Q @ K.T) @ V + Q @ S0[h]
            assert _rel(o_s[:, h], want) < 1e-12, "sequential vs causal linear attention"
            assert _rel(o_c[:, h], want) < 1e-12, "chunked vs causal linear attention"
            Sw = S0[h] + K.T @ V
            assert _rel(S_s[h], Sw) < 1e-12 and _rel(S_c[h], Sw) < 1e-12


def pin_retention_constant_gate(orc):
    """Constant gate g = log(gamma): O = (D * Q K^T) V + diag(gamma^(t+1)) Q S0
    with D[t, m] = gamma^(t-m) for m <= t, else 0 (retention form)."""
    for (T, H, dk, dv, C, gv) in ((70, 2, 8, 8, 16, -0.3), (129, 1, 16, 4, 64, -0.05)):
        q, k, v, g, S0 = _inputs(23 + T, T, H, dk, dv, gate=gv)
        gamma = np.exp(np.float64(np.float32(gv)))
        t = np.arange(T)
        D = np.where(t[:, None] >= t[None, :], gamma ** (t[:, None] - t[None, :]).astype(np.float64), 0.0)
        (o_s, S_s), (o_c, S_c) = _both_forms(orc, q, k, v, g, S0, C)
        for h in range(H):
            Q, K, V = (x[:, h, :].astype(np.float64) for x in (q, k, v))
            want = (D * (Q @ K.T)) @ V + (gamma ** (t + 1))[:, None] * (Q @ S0[h])
            assert _rel(o_s[:, h], want) < 1e-11
            assert _rel(o_c[:, h], want) < 1e-11
            Sw = gamma ** T * S0[h] + (K * (gamma ** (T - 1 - t))[:, None]).T @ V
            assert _rel(S_s[h], Sw) < 1e-11 and _rel(S_c[h], Sw) < 1e-11


def pin_strong_decay(orc):
    """g = -100: the carried state is wiped every token (exp(-100) ~ 4e-44),
    so o_t = (q_t . k_t) v_t to rounding."""
    T, H, dk, dv = 40, 2, 8, 6
    q, k, v, g, S0 = _inputs(5, T, H, dk, dv, gate=-100.0)
    (o_s, _), (o_c, _) = _both_forms(orc, q, k, v, g, S0, 16)
    qk = np.sum(q.astype(np.float64) * k.astype(np.float64), axis=-1, keepdims=True)
    want = qk * v.astype(np.float64)
    assert _rel(o_s, want) < 1e-13 and _rel(o_c, want) < 1e-13


def pin_scale(orc):
    """o is linear in the scale; a power-of-two scale is exact."""
    q, k, v, g, S0 = _inputs(9, 50, 2, 8, 8)
    (o1, _), (c1, _) = _both_forms(orc, q, k, v, g, S0, 16, scale=1.0)
    (o4, _), (c4, _) = _both_forms(orc, q, k, v, g, S0, 16, scale=0.25)
    assert np.array_equal(o4, 0.25 * o1) and np.array_equal(c4, 0.25 * c1)


# -------------------------------------------------- scan: brute force -------
def pin_chunked_equals_sequential(orc):
    """Brute force over tiny shapes: the chunked form equals the recurrence
    (to fp64 rounding), and chunk_states[j] equals the recurrence's state after
    the first j*C tokens."""
    case = 0
    for C in (1, 4, 16, 64):
        for T in sorted({0, 1, 2, C - 1, C, C + 1, 2 * C + 3, 3 * C + 5} - {-1}):
            if T < 0:
                continue
            for (H, dk, dv) in ((1, 1, 1), (2, 4, 16), (1, 16, 4), (2, 8, 8)):
                case += 1
                q, k, v, g, S0 = _inputs(1000 + case, T, H, dk, dv, gate="wide")
                o_s, S_s = orc.sequential(q, k, v, g, S0=S0)
                o_c, cs, S_c = orc.chunked(q, k, v, g, C, S0=S0)
                assert _rel(o_c, o_s) < 1e-12, (C, T, H, dk, dv)
                assert _rel(S_c, S_s) < 1e-12, (C, T, H, dk, dv)
                n = (T + C - 1) // C
                assert cs.shape[0] == n
                for j in range(n):
                    _, Sj = orc.sequential(q[: j * C], k[: j * C], v[: j * C], g[: j * C], S0=S0)
                    assert _rel(cs[j], Sj) < 1e-12, ("chunk state", C, T, j)


def pin_quadratic_single_chunk(orc):
    """T <= C: one chunk, which is the masked quadratic form
    O = (tril(exp(G_i - G_m)) * Q K^T) V + diag(exp(G)) Q S0 with G the
    inclusive cumulative sum of g (built here with numpy cumsum)."""
    T, H, dk, dv, C = 48, 2, 8, 8, 64
    q, k, v, g, S0 = _inputs(77, T, H, dk, dv, gate="wide")
    o_c, _, S_c = orc.chunked(q, k, v, g, C, S0=S0)
    for h in range(H):
        G = np.cumsum(g[:, h].astype(np.float64))
        t = np.arange(T)
        D = np.where(t[:, None] >= t[None, :], np.exp(G[:, None] - G[None, :]), 0.0)
        Q, K, V = (x[:, h, :].astype(np.float64) for x in (q, k, v))
        want = (D * (Q @ K.T)) @ V + np.exp(G)[:, None] * (Q @ S0[h])
        assert _rel(o_c[:, h], want) < 1e-12
        Sw = np.exp(G[-1]) * S0[h] + (K * np.exp(G[-1] - G)[:, None]).T @ V
        assert _rel(S_c[h], Sw) < 1e-12


# ------------------------------------------------------- scan: invariants ---
def pin_composition(orc):
    """Prefill of [0, F) equals prefill of [P', F) started from the state after
    [0, P').  Bitwise for the recurrence at any split, and bitwise for the
    chunked form when P' is a multiple of C (the same chunks are folded by the
    same code) -- the oracle-level form of the paper's restore-then-append
    equation (§5)."""
    T, H, dk, dv, C = 200, 2, 8, 8, 16
    q, k, v, g, S0 = _inputs(31, T, H, dk, dv)
    o_full, S_full = orc.sequential(q, k, v, g, S0=S0)
    for P in (0, 1, 63, 64, 199):
        o_a, S_a = orc.sequential(q[:P], k[:P], v[:P], g[:P], S0=S0)
        o_b, S_b = orc.sequential(q[P:], k[P:], v[P:], g[P:], S0=S_a)
        assert np.array_equal(np.concatenate([o_a, o_b]), o_full)
        assert np.array_equal(S_b, S_full)
    oc_full, cs_full, Sc_full = orc.chunked(q, k, v, g, C, S0=S0)
    for P in (0, 16, 64, 192):
        o_a, _, S_a = orc.chunked(q[:P], k[:P], v[:P], g[:P], C, S0=S0)
        o_b, cs_b, S_b = orc.chunked(q[P:], k[P:], v[P:], g[P:], C, S0=S_a)
        assert np.array_equal(np.concatenate([o_a, o_b]), oc_full)
        assert np.array_equal(S_b, Sc_full)
        assert np.array_equal(cs_b, cs_full[P // C:])


def pin_linearity(orc):
    """(S0, v) -> (2 S0, 2 v) doubles every output and state exactly."""
    q, k, v, g, S0 = _inputs(41, 90, 2, 8, 4)
    (o1, S1), (c1, C1) = _both_forms(orc, q, k, v, g, S0, 16)
    (o2, S2), (c2, C2) = _both_forms(orc, q, k, 2 * v, g, 2 * S0, 16)
    assert np.array_equal(o2, 2 * o1) and np.array_equal(S2, 2 * S1)
    assert np.array_equal(c2, 2 * c1) and np.array_equal(C2, 2 * C1)


def pin_head_permutation(orc):
    """Heads are independent: permuting them permutes the outputs exactly."""
    q, k, v, g, S0 = _inputs(43, 70, 3, 8, 8)
    perm = np.array([2, 0, 1])
    (o1, S1), (c1, C1) = _both_forms(orc, q, k, v, g, S0, 16)
    pq, pk, pv = (np.ascontiguousarray(x[:, perm]) for x in (q, k, v))
    pg = np.ascontiguousarray(g[:, perm])
    (o2, S2), (c2, C2) = _both_forms(orc, pq, pk, pv, pg, S0[perm], 16)
    assert np.array_equal(o2, o1[:, perm]) and np.array_equal(S2, S1[perm])
    assert np.array_equal(c2, c1[:, perm]) and np.array_equal(C2, C1[perm])


def pin_causality(orc):
    """o_t depends on tokens <= t only: changing later tokens leaves earlier
    outputs bit-identical (both forms)."""
    T, H, dk, dv, C = 100, 2, 8, 8, 16
    q, k, v, g, S0 = _inputs(47, T, H, dk, dv)
    (o1, _), (c1, _) = _both_forms(orc, q, k, v, g, S0, C)
    cut = 37
    q2, k2, v2 = q.copy(), k.copy(), v.copy()
    q2[cut:] += 1.0
    k2[cut:] -= 0.5
    v2[cut:] *= 3.0
    g2 = g.copy()
    g2[cut:] -= 0.25
    (o2, _), (c2, _) = _both_forms(orc, q2, k2, v2, g2, S0, C)
    assert np.array_equal(o2[:cut], o1[:cut]) and np.array_equal(c2[:cut], c1[:cut])
    assert not np.array_equal(o2[cut:], o1[cut:])


def pin_outer_product_orientation(orc):
    """With dk != dv the state is dk x dv with S[i, j] accumulating k_i v_j:
    a single token from S0 = 0 gives S = k^T v and o = (q . k) v."""
    q, k, v, g, _ = _inputs(53, 1, 1, 3, 5, gate=0.0)
    o_s, S_s = orc.sequential(q, k, v, g)
    o_c, _, S_c = orc.chunked(q, k, v, g, 4)
    want_S = np.outer(k[0, 0].astype(np.float64), v[0, 0].astype(np.float64))
    assert S_s.shape == (1, 3, 5)
    assert _rel(S_s[0], want_S) < 1e-15 and _rel(S_c[0], want_S) < 1e-15
    want_o = float(np.dot(q[0, 0].astype(np.float64), k[0, 0].astype(np.float64))) * v[0, 0].astype(np.float64)
    assert _rel(o_s[0, 0], want_o) < 1e-14 and _rel(o_c[0, 0], want_o) < 1e-14


SCAN_PINS = [
    pin_counting_scalar, pin_halving_scalar, pin_causal_linear_attention,
    pin_retention_constant_gate, pin_strong_decay, pin_scale,
    pin_chunked_equals_sequential, pin_quadratic_single_chunk, pin_composition,
    pin_linearity, pin_head_permutation, pin_causality, pin_outer_product_orientation,
]


# ----------------------------------------------------------- capsule pins --
def pin_align(orc):
    """P' = floor(P / C) * C (§3 Algorithm 1): a multiple of C, at most P, and
    the re-prefilled remainder P - P' is below C (§5); brute force."""
    for C in range(1, 70):
        for P in range(0, 300):
            Pa = orc.align(P, C)
            assert Pa % C == 0 and Pa <= P < Pa + C, (P, C, Pa)
    # the boundaries of the alignment-stress workload (chunk 64)
    for P, want in ((2048, 2048), (2050, 2048), (2111, 2048), (2112, 2112), (63, 0), (0, 0)):
        assert orc.align(P, 64) == want


def pin_capsule_size_table(orc):
    """Table "capsule breakdown vs prefix" (§7.2) prints capsule sizes 160,
    224, 352 and 608 MB at prefixes 2k, 4k, 8k and 16k: affine in the prefix
    with 64 MB per 2048 tokens.  A set with 32 KiB of positional bytes per
    token and 96 MiB of fixed state reproduces the table exactly when MB is
    read as MiB."""
    tab = np.loadtxt(os.path.join(GOLDEN, "capsule_sizes_tab_break.txt"), comments="#", dtype=np.int64)
    MiB = 1 << 20
    # 16 full-attention layers x {K, V} x 4 heads x d=256 x 1 byte (fp8) per token,
    # 48 recurrent states of 32 x 128 x 128 fp32
    row_bytes = [4 * 256] * 32 + [32 * 128 * 128 * 4] * 48
    rows_total = [16448] * 32 + [1] * 48
    kinds = [0] * 32 + [1] * 48
    for P, mib in tab:
        got = orc.capsule_bytes(row_bytes, rows_total, kinds, orc.align(int(P), 64))
        assert got == int(mib) * MiB, (P, got / MiB, mib)


def _random_set(seed, rows=50):
    """Five host buffers: positional, fixed, positional, fixed, positional."""
    r = rng(seed, 0, "capset")
    bufs, rb, rt, kd = [], [], [], []
    for kind in (0, 1, 0, 1, 0):
        if kind == 0:
            row, nrows = int(r.integers(1, 9)) * 16, rows
        else:
            row, nrows = int(r.integers(1, 40)) * 16, 1
        bufs.append(r.integers(0, 256, size=row * nrows, dtype=np.uint8))
        rb.append(row)
        rt.append(nrows)
        kd.append(kind)
    return bufs, rb, rt, kd


def pin_snapshot_layout(orc):
    """The capsule is the concatenation, in set order, of the first P' rows of
    each positional buffer and all bytes of each fixed buffer (§3
    "Definition": KV valid over [0, P); fixed-size recurrent/conv state)."""
    bufs, rb, rt, kd = _random_set(3)
    for P in (0, 1, 17, 48, 50):
        arena = orc.snapshot(bufs, rb, rt, kd, P)
        parts = [b[: P * r] if k_ == 0 else b for b, r, k_ in zip(bufs, rb, kd)]
        want = np.concatenate(parts) if parts else np.zeros(0, np.uint8)
        assert np.array_equal(arena, want), P
        assert len(arena) == orc.capsule_bytes(rb, rt, kd, P)


def pin_restore_roundtrip(orc):
    """snapshot -> overwrite every live buffer -> restore gives back the
    captured bytes in the valid region; rows at or past P' are not written
    (they are stale and get re-prefilled)."""
    bufs, rb, rt, kd = _random_set(5)
    P = 21
    orig = [b.copy() for b in bufs]
    arena = orc.snapshot(bufs, rb, rt, kd, P)
    for b in bufs:
        b[:] = 0xA5
    orc.restore(arena, bufs, rb, rt, kd, P)
    for b, o, r, k_ in zip(bufs, orig, rb, kd):
        n = P * r if k_ == 0 else len(b)
        assert np.array_equal(b[:n], o[:n])
        assert np.all(b[n:] == 0xA5)


def pin_fork_and_gather(orc):
    """fork(n) = n restores of one capsule; gather gives environment e the
    capsule gallery[ids[e]] (§3 "Four verbs"; §6 episode reset)."""
    bufs, rb, rt, kd = _random_set(7)
    P = 33
    arena = orc.snapshot(bufs, rb, rt, kd, P)
    sets = [[np.zeros_like(b) for b in bufs] for _ in range(3)]
    orc.fork(arena, sets, rb, rt, kd, P)
    for s in sets:
        for b, o, r, k_ in zip(s, bufs, rb, kd):
            n = P * r if k_ == 0 else len(b)
            assert np.array_equal(b[:n], o[:n])
    gallery = []
    for gi in range(4):
        gb, _, _, _ = _random_set(7)
        for b in gb:
            b[:] = (b.astype(np.int64) + gi * 37) % 256
        gallery.append(orc.snapshot(gb, rb, rt, kd, P))
    ids = np.array([3, 0, 3, 1, 2], np.int32)
    envs = [[np.zeros_like(b) for b in bufs] for _ in ids]
    orc.gather(gallery, ids, envs, rb, rt, kd, P)
    for e, i in enumerate(ids):
        assert np.array_equal(orc.snapshot(envs[e], rb, rt, kd, P), gallery[i])
    bad = np.array([0, 4], np.int32)
    try:
        orc.gather(gallery, bad, envs[:2], rb, rt, kd, P)
    except ValueError:
        pass
    else:
        raise AssertionError("out-of-range gallery id accepted")


def pin_digest(orc):
    """64-bit FNV-1a: published test vectors over byte strings
    (fnv1a64_vectors.txt), and the token digest equals the byte digest of the
    ids' little-endian int32 bytes."""
    with open(os.path.join(GOLDEN, "fnv1a64_vectors.txt")) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            text, hexval = line.rsplit(None, 1)
            text = text.strip()
            assert text[0] == text[-1] == '"'
            text = text[1:-1]
            assert orc.digest_bytes(text.encode()) == int(hexval, 16), (text, hexval)
    ids = np.array([0, 1, 151935, 7, -1], np.int32)
    assert orc.digest_tokens(ids) == orc.digest_bytes(ids.astype("<i4").tobytes())
    assert orc.digest_tokens(ids[:0]) == int("cbf29ce484222325", 16)


def pin_append_history(orc):
    """Append of a suffix, brute force: a positional buffer equals the token
    history written row by row at its positions; a fixed window equals the
    last W rows of its full history (initial rows, then every appended row),
    for suffixes shorter than, equal to and longer than the window; buffers
    without a source keep their bytes; a positional overflow copies nothing."""
    r = rng(21, 0, "appendpin")
    rb_pos, rows_pos, rb_win, W = 48, 40, 32, 4
    kinds = [0, 1, 1]
    rbs, rts = [rb_pos, rb_win, 64], [rows_pos, W, 2]
    pos_buf = r.integers(0, 256, rows_pos * rb_pos, dtype=np.uint8)
    win_buf = r.integers(0, 256, W * rb_win, dtype=np.uint8)
    fixed = r.integers(0, 256, 128, dtype=np.uint8)
    fixed0 = fixed.copy()
    pos_hist = pos_buf.reshape(rows_pos, rb_pos).copy()
    win_hist = list(win_buf.reshape(W, rb_win).copy())
    position = 5
    for n in (1, 2, 4, 7, 1, 3):
        src_pos = r.integers(0, 256, n * rb_pos, dtype=np.uint8)
        src_win = r.integers(0, 256, n * rb_win, dtype=np.uint8)
        assert orc.append([pos_buf, win_buf, fixed], [src_pos, src_win, None], rbs, rts, kinds, position, n) == 0
        pos_hist[position:position + n] = src_pos.reshape(n, rb_pos)
        win_hist.extend(src_win.reshape(n, rb_win))
        position += n
        assert np.array_equal(pos_buf.reshape(rows_pos, rb_pos), pos_hist)
        assert np.array_equal(win_buf.reshape(W, rb_win), np.stack(win_hist[-W:]))
        assert np.array_equal(fixed, fixed0)
    before = pos_buf.copy(), win_buf.copy()
    src_pos = r.integers(0, 256, 20 * rb_pos, dtype=np.uint8)
    src_win = r.integers(0, 256, 20 * rb_win, dtype=np.uint8)
    assert orc.append([pos_buf, win_buf, fixed], [src_pos, src_win, None], rbs, rts, kinds, 30, 20) == -1
    assert np.array_equal(pos_buf, before[0]) and np.array_equal(win_buf, before[1])


CAPSULE_PINS = [pin_align, pin_capsule_size_table, pin_snapshot_layout,
                pin_restore_roundtrip, pin_fork_and_gather, pin_digest, pin_append_history]


# ------------------------------------------------------------- FP8 KV ----
# OCP 8-bit floating point, E4M3 ("E4M3FN"): the format's published facts,
# and torch's own float8_e4m3fn / bfloat16 conversions (an implementation
# independent of the oracle) over the range where both define the result.
def pin_e4m3_published_values(orc):
    """Largest finite 448 = S.1111.110, smallest normal 2^-6 = 0.0001.000,
    smallest subnormal 2^-9, largest subnormal 7/8 * 2^-6, one = 0.0111.000,
    NaN = S.1111.111, no infinities; the negative half mirrors the positive."""
    assert orc.e4m3_decode(0x7E) == 448.0
    assert orc.e4m3_decode(0x08) == 2.0 ** -6
    assert orc.e4m3_decode(0x01) == 2.0 ** -9
    assert orc.e4m3_decode(0x07) == 0.875 * 2.0 ** -6
    assert orc.e4m3_decode(0x38) == 1.0
    assert np.isnan(orc.e4m3_decode(0x7F)) and np.isnan(orc.e4m3_decode(0xFF))
    vals = [orc.e4m3_decode(c) for c in range(0x7F)]
    assert all(np.isfinite(vals)) and all(b > a for a, b in zip(vals, vals[1:]))   # strictly increasing
    for c in range(0x7F):
        assert orc.e4m3_decode(c | 0x80) == -orc.e4m3_decode(c) or c == 0


def pin_e4m3_against_torch(orc):
    """Every code decodes as torch's float8_e4m3fn does; encoding agrees with
    torch's round-to-nearest-even cast on |x| < 464 (beyond that torch gives
    NaN, the oracle saturates to 448 -- the reading taken)."""
    import torch
    codes = np.arange(256, dtype=np.uint8)
    tv = torch.from_numpy(codes).view(torch.float8_e4m3fn).float().numpy()
    for c in range(256):
        ov = orc.e4m3_decode(c)
        assert (np.isnan(ov) and np.isnan(tv[c])) or ov == tv[c], c
    r = rng(11, 0, "fp8pin")
    xs = np.concatenate([r.standard_normal(3000) * 10.0, r.uniform(-463.9, 463.9, 2000),
                         r.standard_normal(2000) * 2.0 ** -8,
                         (np.array([tv[c] for c in range(0x7E)]) + np.array([tv[c + 1] for c in range(0x7E)])) / 2,
                         -(np.array([tv[c] for c in range(0x7E)]) + np.array([tv[c + 1] for c in range(0x7E)])) / 2])
    xs = xs.astype(np.float32)
    want = torch.from_numpy(xs).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    for x, w in zip(xs, want):
        assert orc.e4m3_encode(x) == w, (float(x), orc.e4m3_encode(x), int(w))


def pin_e4m3_round_trip_and_saturation(orc):
    """encode(decode(c)) = c for every finite code; values at or beyond 448
    (and +-inf) saturate to +-448; NaN keeps its sign; the error of a
    normal-range value is at most half a unit in the last place: 2^-4 relative."""
    for c in range(256):
        if (c & 0x7F) == 0x7F:
            continue
        assert orc.e4m3_encode(orc.e4m3_decode(c)) == c, c
    for x, want in [(448.0, 0x7E), (449.0, 0x7E), (1e30, 0x7E), (float("inf"), 0x7E),
                    (-1e30, 0xFE), (float("-inf"), 0xFE), (float("nan"), 0x7F), (-float("nan"), 0xFF)]:
        assert orc.e4m3_encode(x) == want, (x, want)
    r = rng(12, 0, "fp8pin")
    xs = (r.uniform(2.0 ** -6, 440.0, 4000) * r.choice([-1.0, 1.0], 4000)).astype(np.float32)
    for x in xs:
        y = orc.e4m3_decode(orc.e4m3_encode(x))
        assert abs(y - float(x)) <= abs(float(x)) * 2.0 ** -4, (float(x), y)


def pin_fp8_arrays_scale_and_bf16(orc):
    """The array forms apply the scale (stored value x / scale, restored
    value code * scale), rounding to bf16 as torch's float -> bfloat16 cast
    does (round to nearest even)."""
    import torch
    r = rng(13, 0, "fp8pin")
    x = r.standard_normal(4096).astype(np.float32) * 3.0
    bits = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    xb = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).float().numpy()
    for scale in (1.0, 0.03125, 2.5):
        q = orc.fp8_quantize(bits, scale)
        inv = np.float32(1.0) / np.float32(scale)
        tq = torch.from_numpy((xb * inv).astype(np.float32)).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
        sat = np.abs(xb * inv) >= 448.0
        assert np.array_equal(q[~sat], tq[~sat]), scale
        assert np.all(q[sat & (xb > 0)] == 0x7E) and np.all(q[sat & (xb < 0)] == 0xFE)
        d = orc.fp8_dequantize(q, scale)
        fv = torch.from_numpy(q).view(torch.float8_e4m3fn).float().numpy() * np.float32(scale)
        td = torch.from_numpy(fv.astype(np.float32)).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
        assert np.array_equal(d, td), scale
    ys = r.standard_normal(20000).astype(np.float32) * np.float32(2.0) ** r.integers(-20, 20, 20000).astype(np.float32)
    # exact midpoints between neighbouring bf16 values: ties go to the even one
    base = (r.integers(0x0080, 0x7F00, 2000).astype(np.uint32) << 16) | (r.integers(0, 2, 2000).astype(np.uint32) << 31)
    mids = (base | 0x8000).view(np.float32)
    ys = np.concatenate([ys[:3000], mids])
    tb = torch.from_numpy(ys).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    for y, w in zip(ys, tb):
        assert orc.bf16_round(y) == w, (float(y), orc.bf16_round(y), int(w))


# ------------------------------------------------------- gated delta rule ----
def _gdn_inputs(seed, T, H, dk, dv, g_lo=-0.3):
    r = rng(seed, 0, "gdnpin")
    q = r.standard_normal((T, H, dk)).astype(np.float32)
    k = r.standard_normal((T, H, dk))
    k = (k / np.linalg.norm(k, axis=-1, keepdims=True)).astype(np.float32)
    v = r.standard_normal((T, H, dv)).astype(np.float32)
    g = r.uniform(g_lo, 0.0, (T, H)).astype(np.float32)
    beta = r.uniform(0.0, 1.0, (T, H)).astype(np.float32)
    S0 = r.standard_normal((H, dk, dv))
    return q, k, v, g, beta, S0


def pin_gdn_chunked_equals_sequential(orc):
    """Two algorithms: the chunked WY form equals the recurrence (any chunk
    size, ragged tail, entering state), and its chunk states are the
    recurrence's states at the chunk starts."""
    q, k, v, g, b, S0 = _gdn_inputs(1, 150, 2, 16, 8)
    o1, s1 = orc.gdn_sequential(q, k, v, g, b, S0, scale=0.5)
    for C in (1, 7, 64):
        o2, cs, s2 = orc.gdn_chunked(q, k, v, g, b, C, S0, scale=0.5)
        assert _rel(o2, o1) < 1e-11 and _rel(s2, s1) < 1e-11, C
        for j in range(1, cs.shape[0]):
            _, sj = orc.gdn_sequential(q[: j * C], k[: j * C], v[: j * C], g[: j * C], b[: j * C], S0)
            assert _rel(cs[j], sj) < 1e-11, (C, j)


def pin_gdn_beta_zero_is_pure_decay(orc):
    """beta = 0 writes nothing: S_t = exp(G_t) S0, o_t = exp(G_t) q_t S0."""
    q, k, v, g, b, S0 = _gdn_inputs(2, 70, 2, 8, 4, g_lo=-1.0)
    b[:] = 0.0
    G = np.cumsum(g.astype(np.float64), axis=0)
    want_o = np.exp(G)[:, :, None] * np.einsum("thd,hde->the", q.astype(np.float64), S0)
    for o, S in (orc.gdn_sequential(q, k, v, g, b, S0), orc.gdn_chunked(q, k, v, g, b, 16, S0)[::2]):
        assert _rel(o, want_o) < 1e-12
        assert _rel(S, np.exp(G[-1])[:, None, None] * S0) < 1e-12


def pin_gdn_orthonormal_keys_store_values(orc):
    """With orthonormal keys and beta = 1 the delta rule stores each value
    exactly under its key: right after token t, k_t S_t = v_t; an earlier key
    reads its value decayed by the gates since, k_i S_t = exp(G_t - G_i) v_i;
    directions orthogonal to every key keep exp(G_t) S0."""
    r = rng(3, 0, "gdnpin")
    dk, dv, n = 16, 5, 6
    Hm = np.array([[1.0]])
    while Hm.shape[0] < dk:                            # Sylvester's Hadamard matrix
        Hm = np.block([[Hm, Hm], [Hm, -Hm]])
    Qm = Hm[r.permutation(dk)] / 4.0                   # orthonormal rows, exact in fp32
    keys = Qm[:n].astype(np.float32)
    free = Qm[n:]                                      # their complement
    k = keys[:, None, :]
    v = r.standard_normal((n, 1, dv)).astype(np.float32)
    g = r.uniform(-0.5, 0.0, (n, 1)).astype(np.float32)
    b = np.ones((n, 1), np.float32)
    S0 = r.standard_normal((1, dk, dv))
    G = np.cumsum(g[:, 0].astype(np.float64))
    kd = keys.astype(np.float64)
    for t in range(n):
        for fn in (lambda T: orc.gdn_sequential(k[:T], k[:T], v[:T], g[:T], b[:T], S0)[1],
                   lambda T: orc.gdn_chunked(k[:T], k[:T], v[:T], g[:T], b[:T], 4, S0)[2]):
            S = fn(t + 1)[0]
            for i in range(t + 1):
                want = np.exp(G[t] - G[i]) * v[i, 0].astype(np.float64)
                assert np.abs(kd[i] @ S - want).max() < 1e-9, (t, i)
            assert np.abs(free @ S - np.exp(G[t]) * (free @ S0[0])).max() < 1e-9


def pin_gdn_linearity_and_causality(orc):
    """(o, S) is linear in (v, S0) jointly for fixed q, k, g, beta; outputs
    before a token do not depend on it or anything after it."""
    q, k, v1, g, b, S1 = _gdn_inputs(4, 90, 1, 8, 4)
    _, _, v2, _, _, S2 = _gdn_inputs(5, 90, 1, 8, 4)
    o1, s1 = orc.gdn_chunked(q, k, v1, g, b, 32, S1)[::2]
    o2, s2 = orc.gdn_chunked(q, k, v2, g, b, 32, S2)[::2]
    v3 = (2.0 * v1.astype(np.float64) - 3.0 * v2.astype(np.float64)).astype(np.float32)
    o3, s3 = orc.gdn_chunked(q, k, v3, g, b, 32, 2.0 * S1 - 3.0 * S2)[::2]
    dv_err = (v3.astype(np.float64) - (2.0 * v1.astype(np.float64) - 3.0 * v2.astype(np.float64)))
    assert np.abs(dv_err).max() < 1e-5  # v3 is the fp32 rounding of the combination
    o12, s12 = orc.gdn_sequential(q, k, v3, g, b, 2.0 * S1 - 3.0 * S2)
    assert _rel(o3, o12) < 1e-11 and _rel(s3, s12) < 1e-11
    oL = 2.0 * o1 - 3.0 * o2
    assert _rel(o3, oL) < 1e-5 and _rel(s3, 2.0 * s1 - 3.0 * s2) < 1e-5
    cut = 50
    k2, v4 = k.copy(), v1.copy()
    k2[cut:] = np.roll(k2[cut:], 1, axis=-1)
    v4[cut:] *= -2.0
    o4 = orc.gdn_chunked(q, k2, v4, g, b, 32, S1)[0]
    assert np.array_equal(o4[:cut], o1[:cut]) and not np.allclose(o4[cut:], o1[cut:])


GDN_PINS = [pin_gdn_chunked_equals_sequential, pin_gdn_beta_zero_is_pure_decay,
            pin_gdn_orthonormal_keys_store_values, pin_gdn_linearity_and_causality]

FP8_PINS = [pin_e4m3_published_values, pin_e4m3_against_torch, pin_e4m3_round_trip_and_saturation,
            pin_fp8_arrays_scale_and_bf16]

ALL_PINS = SCAN_PINS + CAPSULE_PINS + FP8_PINS + GDN_PINS
