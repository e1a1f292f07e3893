"""Capsule verbs on the GPU (through the C ABI) against the oracle's memcpy
semantics: capsule bytes and restored live bytes must be identical."""
import numpy as np
import pytest

import paper_2606_20537_amd as cap
from gpu_util import device_bytes

pytestmark = pytest.mark.gpu

# A small hybrid-like set: positional K/V rows of 4 heads x 64 bf16, recurrent
# states, conv tails -- interleaved so every buffer kind sits between others.
LAYOUT = [
    ("kv0.k", 512, 300, cap.CAP_KIND_POSITIONAL),
    ("lin0.state", 2 * 64 * 64 * 4, 1, cap.CAP_KIND_FIXED),
    ("kv0.v", 512, 300, cap.CAP_KIND_POSITIONAL),
    ("lin0.conv", 4 * 256 * 2, 1, cap.CAP_KIND_FIXED),
    ("kv1.k", 64 * 1024, 300, cap.CAP_KIND_POSITIONAL),     # rows wider than a copy tile
    ("lin1.state", 16, 1, cap.CAP_KIND_FIXED),               # a single 16-byte vector
    ("kv1.v", 48, 300, cap.CAP_KIND_POSITIONAL),             # rows of 3 vectors
]
CHUNK = 64
KEY = 0xD15EA5E


def _make_set(seed, layout=LAYOUT, key=KEY):
    bufs = []
    for i, (name, rb, rows, kind) in enumerate(layout):
        bufs.append((name, device_bytes(rb * rows, seed=seed * 100 + i, name=name), rb, rows, kind))
    s = cap.cap_set_create(bufs, CHUNK, key)
    return s, bufs


def _host(bufs):
    return [b[1].cpu().numpy() for b in bufs]


def _lay(bufs):
    return [b[2] for b in bufs], [b[3] for b in bufs], [b[4] for b in bufs]


@pytest.mark.parametrize("P", [0, 63, 64, 130, 192, 300])
def test_snapshot_bytes_match_oracle(orc, P):
    import torch
    s, bufs = _make_set(1)
    Pa = cap.cap_align_boundary(P, CHUNK)
    cap.cap_set_set_position(s, Pa)
    nbytes = cap.capsule_bytes(s, P)
    rb, rt, kd = _lay(bufs)
    assert nbytes == orc.capsule_bytes(rb, rt, kd, Pa)
    arena = device_bytes(nbytes + 4096, fill=0xEE)
    c = cap.capsule_snapshot(s, P, 42, arena)
    torch.cuda.synchronize()
    want = orc.snapshot(_host(bufs), rb, rt, kd, Pa)
    got = arena.cpu().numpy()
    assert np.array_equal(got[:nbytes], want)
    assert np.all(got[nbytes:] == 0xEE)  # nothing written past the capsule
    info = cap.capsule_info(c)
    assert info["P_aligned"] == Pa and info["bytes"] == nbytes and info["prefix_digest"] == 42


def test_restore_after_poison_is_byte_exact(orc):
    """Dirtied-state check (§5): every live byte overwritten before restore."""
    import torch
    s, bufs = _make_set(2)
    P = 150
    Pa = cap.cap_align_boundary(P, CHUNK)
    cap.cap_set_set_position(s, Pa)
    orig = _host(bufs)
    arena = device_bytes(cap.capsule_bytes(s, P))
    c = cap.capsule_snapshot(s, P, 7, arena)
    for b in bufs:
        b[1].fill_(0xFF)
    cap.cap_set_set_position(s, 0)
    assert cap.capsule_restore(c, s, 7) == Pa
    assert cap.cap_set_get_position(s) == Pa
    torch.cuda.synchronize()
    rb, rt, kd = _lay(bufs)
    want = [o.copy() for o in orig]
    for w in want:
        w[:] = 0xFF
    orc.restore(orc.snapshot(orig, rb, rt, kd, Pa), want, rb, rt, kd, Pa)
    for got, w in zip(_host(bufs), want):
        assert np.array_equal(got, w)


def test_fork_writes_every_branch(orc):
    import torch
    src, bufs = _make_set(3)
    P = 256
    cap.cap_set_set_position(src, P)
    arena = device_bytes(cap.capsule_bytes(src, P))
    c = cap.capsule_snapshot(src, P, 9, arena)
    branches = [_make_set(10 + i) for i in range(5)]
    cap.capsule_fork(c, [b[0] for b in branches], 9)
    torch.cuda.synchronize()
    rb, rt, kd = _lay(bufs)
    want = orc.snapshot(_host(bufs), rb, rt, kd, P)
    for s, bb in branches:
        assert np.array_equal(orc.snapshot(_host(bb), rb, rt, kd, P), want)
        assert cap.cap_set_get_position(s) == P


def test_gather_restore_matches_oracle(orc):
    import torch
    P = 192
    gallery, gsets = [], []
    for gi in range(5):
        s, bufs = _make_set(20 + gi)
        cap.cap_set_set_position(s, P)
        arena = device_bytes(cap.capsule_bytes(s, P))
        gallery.append(cap.capsule_snapshot(s, P, 0, arena))
        gsets.append((s, bufs))
    envs = [_make_set(40 + e) for e in range(9)]
    ids = np.random.default_rng(5).integers(0, 5, size=9).astype(np.int32)
    cap.capsule_gather_restore(gallery, ids, [e[0] for e in envs])
    torch.cuda.synchronize()
    rb, rt, kd = _lay(gsets[0][1])
    for (s, bb), i in zip(envs, ids):
        assert np.array_equal(orc.snapshot(_host(bb), rb, rt, kd, P),
                              gallery[i].arena_ref.cpu().numpy()[: cap.capsule_info(gallery[i])["bytes"]])


def test_errors_enqueue_nothing():
    """Digest, deployment key, layout, state and size errors return before any
    device write: the live buffers keep their bytes."""
    import torch
    s, bufs = _make_set(4)
    cap.cap_set_set_position(s, 128)
    arena = device_bytes(cap.capsule_bytes(s, 128))
    c = cap.capsule_snapshot(s, 128, 1234, arena)
    torch.cuda.synchronize()
    for b in bufs:
        b[1].fill_(0x5A)
    before = _host(bufs)

    def code(fn, *a):
        try:
            fn(*a)
        except cap.CapsuleError as e:
            return e.status
        return cap.CAP_OK

    assert code(cap.capsule_restore, c, s, 999) == cap.CAP_E_DIGEST
    other_key, _ = _make_set(5, key=KEY + 1)
    assert code(cap.capsule_restore, c, other_key, 1234) == cap.CAP_E_DIGEST
    other_layout, _ = _make_set(6, layout=LAYOUT[:-1])
    assert code(cap.capsule_restore, c, other_layout, 1234) == cap.CAP_E_SIZE
    assert code(cap.capsule_fork, c, [s, s], 1234) == cap.CAP_E_INVAL
    small = device_bytes(16)
    assert code(cap.capsule_snapshot, s, 128, 0, small) == cap.CAP_E_SIZE
    assert code(cap.capsule_snapshot, s, 200, 0, arena) == cap.CAP_E_STATE  # position 128 != 192
    assert code(cap.cap_set_set_position, s, 301) == cap.CAP_E_SIZE
    assert code(cap.capsule_gather_restore, [c], [1], [s]) == cap.CAP_E_INVAL
    torch.cuda.synchronize()
    for got, b in zip(_host(bufs), before):
        assert np.array_equal(got, b)


def test_rollback_to_earlier_capsule():
    """rollback = restore of an earlier capsule of the same session (§3)."""
    import torch
    s, bufs = _make_set(7)
    cap.cap_set_set_position(s, 64)
    a1 = device_bytes(cap.capsule_bytes(s, 64))
    c1 = cap.capsule_snapshot(s, 64, 1, a1)
    at64 = _host(bufs)
    for b in bufs:
        b[1].add_(1)
    cap.cap_set_set_position(s, 256)
    a2 = device_bytes(cap.capsule_bytes(s, 256))
    cap.capsule_snapshot(s, 256, 2, a2)
    cap.capsule_restore(c1, s, 1)
    torch.cuda.synchronize()
    for got, w, (_, _, rb, rows, kind) in zip(_host(bufs), at64, bufs):
        n = 64 * rb if kind == cap.CAP_KIND_POSITIONAL else rb * rows
        assert np.array_equal(got[:n], w[:n])


def test_explicit_release_then_collection_is_safe():
    """Releasing a capsule (or destroying a set) through the module functions
    and then dropping the Python object frees each C handle once: a new
    capsule made afterwards (which may reuse the freed header's memory)
    still restores byte for byte."""
    import gc
    import torch
    s, bufs = _make_set(9)
    cap.cap_set_set_position(s, 192)
    nbytes = cap.capsule_bytes(s, 192)
    arena = device_bytes(nbytes, fill=0)
    for rnd in range(3):
        c = cap.capsule_snapshot(s, 192, 7, arena)
        cap.capsule_release(c)
        assert c.handle is None
        cap.capsule_release(c)   # a second release is a no-op
        del c
        gc.collect()
    c = cap.capsule_snapshot(s, 192, 7, arena)
    want = [b[1].clone() for b in bufs]
    for b in bufs:
        b[1].fill_(0x5A)
    cap.capsule_restore(c, s, 7)
    torch.cuda.synchronize()
    for b, w in zip(bufs, want):
        n = b[2] * (192 if b[4] == cap.CAP_KIND_POSITIONAL else b[3])
        assert torch.equal(b[1][:n], w[:n]), b[0]
    s2, _ = _make_set(10)
    cap.cap_set_destroy(s2)
    assert s2.handle is None
    s2.destroy()                 # no-op
    del s2
    gc.collect()


def test_overlapping_destination_sets_are_rejected():
    """Two live sets over the same device buffers: a gather writing different
    capsules into them would race, and a fork would write the same bytes
    twice -- both are CAP_E_INVAL before anything is enqueued."""
    import torch
    s_a, bufs = _make_set(21)
    s_b = cap.cap_set_create(bufs, CHUNK, KEY)          # the same buffers, another handle
    s_c, _ = _make_set(22)
    P = 128
    cap.cap_set_set_position(s_a, P)
    arena = device_bytes(cap.capsule_bytes(s_a, P), fill=0)
    c = cap.capsule_snapshot(s_a, P, 5, arena)
    torch.cuda.synchronize()
    before = [b[1].clone() for b in bufs]
    for call in (lambda: cap.capsule_gather_restore([c], [0, 0], [s_b, s_a]),
                 lambda: cap.capsule_fork(c, [s_c, s_b, s_a], 5)):
        with pytest.raises(cap.CapsuleError) as ei:
            call()
        assert ei.value.status == cap.CAP_E_INVAL
    torch.cuda.synchronize()
    for b, x in zip(bufs, before):
        assert torch.equal(b[1], x)
    cap.capsule_fork(c, [s_c, s_b], 5)                    # disjoint destinations are fine


def test_rejected_arena_keeps_the_callers_pending_error():
    """An arena the device cannot address is CAP_E_INVAL; the library clears
    the error its own pointer query raised only when none was pending, so an
    error the caller left pending stays pending."""
    import ctypes as ct
    import torch
    hip = ct.CDLL("libamdhip64.so")
    hip.hipGetLastError.restype = ct.c_int
    hip.hipPeekAtLastError.restype = ct.c_int
    hip.hipSetDevice.argtypes = [ct.c_int]
    s, bufs = _make_set(31)
    P = 64
    cap.cap_set_set_position(s, P)
    pageable = np.zeros(cap.capsule_bytes(s, P) + 64, np.uint8)
    addr = (pageable.ctypes.data + 15) & ~15
    torch.cuda.synchronize()
    assert hip.hipGetLastError() == 0
    # nothing pending: the query's own error is cleared
    with pytest.raises(cap.CapsuleError) as ei:
        cap.capsule_snapshot(s, P, 0, addr, arena_bytes=cap.capsule_bytes(s, P))
    assert ei.value.status == cap.CAP_E_INVAL
    assert hip.hipPeekAtLastError() == 0
    # does the runtime keep an error pending across a successful call?
    dev = ct.c_int(-1)
    hip.hipGetDevice.argtypes = [ct.POINTER(ct.c_int)]
    assert hip.hipSetDevice(1 << 20) != 0                  # an invalid device index: a host-side error
    assert hip.hipGetDevice(ct.byref(dev)) == 0
    sticky = hip.hipPeekAtLastError() != 0
    hip.hipGetLastError()
    if not sticky:
        print("this runtime clears the stored error on every successful call; nothing can stay pending")
        return
    # an error left pending by the caller survives the call
    assert hip.hipSetDevice(1 << 20) != 0
    with pytest.raises(cap.CapsuleError):
        cap.capsule_snapshot(s, P, 0, addr, arena_bytes=cap.capsule_bytes(s, P))
    assert hip.hipPeekAtLastError() != 0
    assert hip.hipGetLastError() != 0                      # cleared here, by the caller
    assert hip.hipGetLastError() == 0


def test_append_across_two_launches_matches_oracle(orc):
    """An append to 200 buffers takes two launches (128 buffers each at most);
    every row lands where the oracle's append puts it."""
    import torch
    layout = [("p%d" % i, 32 * (1 + i % 3), 40, cap.CAP_KIND_POSITIONAL) for i in range(150)]
    layout += [("w%d" % i, 64, 4, cap.CAP_KIND_FIXED) for i in range(50)]
    s, bufs = _make_set(41, layout)
    pos, n = 7, 5
    cap.cap_set_set_position(s, pos)
    srcs = [device_bytes(n * rb, seed=4100 + i, name="src%d" % i) for i, (_, rb, _, _) in enumerate(layout)]
    host = _host(bufs)
    cap.cap_set_append(s, srcs, n)
    torch.cuda.synchronize()
    rb, rt, kd = _lay(bufs)
    assert orc.append(host, [x.cpu().numpy() for x in srcs], rb, rt, kd, pos, n) == 0
    for b, want in zip(bufs, host):
        assert np.array_equal(b[1].cpu().numpy(), want), b[0]
    assert cap.cap_set_get_position(s) == pos + n


def _big_layout(n, seed):
    """n buffers of mixed kinds and widths (positional rows of 16-80 B over
    200 rows, fixed buffers of 16-272 B), in a seeded order."""
    rng = np.random.default_rng(seed)
    out = []
    for i in range(n):
        if rng.random() < 0.5:
            out.append(("p%d" % i, 16 * int(rng.integers(1, 6)), 200, cap.CAP_KIND_POSITIONAL))
        else:
            out.append(("f%d" % i, 16 * int(rng.integers(1, 18)), 1, cap.CAP_KIND_FIXED))
    return out


def test_snapshot_restore_with_the_maximum_buffer_count(orc):
    """A set of CAP_MAX_BUFFERS (512) buffers, the largest segment table a
    copy block holds: snapshot bytes equal the oracle's, and restore after
    poisoning rewrites exactly the capsule's bytes (rows past P' untouched)."""
    import torch
    layout = _big_layout(cap.CAP_MAX_BUFFERS, 1)
    s, bufs = _make_set(60, layout)
    P = 140
    Pa = cap.cap_align_boundary(P, CHUNK)
    cap.cap_set_set_position(s, Pa)
    orig = _host(bufs)
    rb, rt, kd = _lay(bufs)
    nbytes = cap.capsule_bytes(s, P)
    assert nbytes == orc.capsule_bytes(rb, rt, kd, Pa)
    arena = device_bytes(nbytes)
    c = cap.capsule_snapshot(s, P, 3, arena)
    torch.cuda.synchronize()
    assert np.array_equal(arena.cpu().numpy(), orc.snapshot(orig, rb, rt, kd, Pa))
    for b in bufs:
        b[1].fill_(0xA5)
    assert cap.capsule_restore(c, s, 3) == Pa
    torch.cuda.synchronize()
    want = [np.full_like(o, 0xA5) for o in orig]
    orc.restore(orc.snapshot(orig, rb, rt, kd, Pa), want, rb, rt, kd, Pa)
    for got, w in zip(_host(bufs), want):
        assert np.array_equal(got, w)


def test_fork_to_the_maximum_destination_count_over_two_launches(orc):
    """Fork into CAP_MAX_FORK (16) sets of 200 buffers: 3,200 destination
    pointers exceed one launch's LDS table, so the call takes two launches;
    every branch holds the capsule's bytes and nothing else changed."""
    import torch
    layout = _big_layout(200, 2)
    src, bufs = _make_set(70, layout)
    P = 128
    cap.cap_set_set_position(src, P)
    arena = device_bytes(cap.capsule_bytes(src, P))
    c = cap.capsule_snapshot(src, P, 5, arena)
    branches = [_make_set(80 + i, layout) for i in range(cap.CAP_MAX_FORK)]
    before = [_host(bb) for _, bb in branches]
    cap.capsule_fork(c, [b[0] for b in branches], 5)
    torch.cuda.synchronize()
    rb, rt, kd = _lay(bufs)
    snap = orc.snapshot(_host(bufs), rb, rt, kd, P)
    for (s, bb), old in zip(branches, before):
        want = [o.copy() for o in old]
        orc.restore(snap, want, rb, rt, kd, P)
        for got, w in zip(_host(bb), want):
            assert np.array_equal(got, w)
        assert cap.cap_set_get_position(s) == P


def test_gather_over_more_environments_than_one_launch(orc):
    """70 environments from a gallery of 3 capsules: the call takes two
    launches (64 + 6 environments); each environment holds its capsule's
    bytes and nothing else changed."""
    import torch
    P = 64
    gallery = []
    for gi in range(3):
        s, bufs = _make_set(90 + gi)
        cap.cap_set_set_position(s, P)
        arena = device_bytes(cap.capsule_bytes(s, P))
        gallery.append((cap.capsule_snapshot(s, P, 0, arena), _host(bufs)))
    envs = [_make_set(100 + e) for e in range(70)]
    before = [_host(bb) for _, bb in envs]
    ids = np.random.default_rng(9).integers(0, 3, size=70).astype(np.int32)
    cap.capsule_gather_restore([g[0] for g in gallery], ids, [e[0] for e in envs])
    torch.cuda.synchronize()
    rb, rt, kd = _lay(envs[0][1])
    for (s, bb), old, i in zip(envs, before, ids):
        want = [o.copy() for o in old]
        orc.restore(orc.snapshot(gallery[i][1], rb, rt, kd, P), want, rb, rt, kd, P)
        for got, w in zip(_host(bb), want):
            assert np.array_equal(got, w)
        assert cap.cap_set_get_position(s) == P
