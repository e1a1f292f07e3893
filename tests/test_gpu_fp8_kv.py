"""FP8 KV region on the GPU through the C ABI against the oracle, bit for bit
(§3 "Definition": FP8-KV roughly halves the capsule; §3 cost model: the BF16
working stage is rebuilt lazily after a restore).  Every bf16 input pattern
and every E4M3 code is converted; multi-segment launches cover ragged
segment sizes; an FP8-KV live set goes through snapshot / poison / restore /
stage rebuild and must equal the cold path's stage."""
import numpy as np
import pytest

import paper_2606_20537_amd as cap
from gpu_util import device_bytes

pytestmark = pytest.mark.gpu

SCALES = [1.0, 0.015625, 3.0, 0.3]


def _all_bf16():
    return np.arange(65536, dtype=np.uint32).astype(np.uint16)


@pytest.mark.parametrize("scale", SCALES)
def test_quantize_every_bf16_pattern(orc, scale):
    import torch
    bits = _all_bf16()
    src = torch.from_numpy(bits.view(np.int16)).cuda()
    dst = torch.full((bits.size,), 0xAA, dtype=torch.uint8, device="cuda")
    cap.kv_fp8_quantize([(src, dst, bits.size, scale)])
    torch.cuda.synchronize()
    got = dst.cpu().numpy()
    want = orc.fp8_quantize(bits, scale)
    bad = np.nonzero(got != want)[0]
    assert bad.size == 0, [(hex(int(bits[i])), int(got[i]), int(want[i])) for i in bad[:8]]


@pytest.mark.parametrize("scale", SCALES + [1e30])
def test_dequantize_every_code(orc, scale):
    import torch
    codes = np.tile(np.arange(256, dtype=np.uint16).astype(np.uint8), 16)
    src = torch.from_numpy(codes).cuda()
    dst = torch.zeros(codes.size, dtype=torch.int16, device="cuda")
    cap.kv_fp8_dequantize([(src, dst, codes.size, scale)])
    torch.cuda.synchronize()
    got = dst.cpu().numpy().view(np.uint16)
    want = orc.fp8_dequantize(codes, scale)
    bad = np.nonzero(got != want)[0]
    assert bad.size == 0, [(int(codes[i]), hex(int(got[i])), hex(int(want[i]))) for i in bad[:8]]


def test_segments_in_one_launch(orc):
    """Ragged segment sizes (one group, a block plus one group, an empty
    segment, a large one) convert independently in a single launch, and
    nothing is written past any segment."""
    import torch
    sizes = [16, 8192 + 16, 0, 48, 1 << 20, 4096]
    scales = [1.0, 0.25, 1.0, 2.0, 0.0625, 1.5]
    rng = np.random.default_rng(5)
    segs, refs, bufs = [], [], []
    for n, sc in zip(sizes, scales):
        x = (rng.standard_normal(n) * 4).astype(np.float32)
        bits = torch.from_numpy(x).to(torch.bfloat16).view(torch.int16)
        src = bits.cuda()
        dst = torch.full((n + 64,), 0xEE, dtype=torch.uint8, device="cuda")
        segs.append((src, dst, n, sc))
        refs.append(orc.fp8_quantize(bits.numpy().view(np.uint16), sc))
        bufs.append(dst)
    cap.kv_fp8_quantize(segs)
    back = [torch.full((n + 32,), 0x7777, dtype=torch.int16, device="cuda") for n in sizes]
    cap.kv_fp8_dequantize([(b, bk, n, sc) for b, bk, n, sc in zip(bufs, back, sizes, scales)])
    torch.cuda.synchronize()
    for n, sc, ref, b, bk in zip(sizes, scales, refs, bufs, back):
        got = b.cpu().numpy()
        assert np.array_equal(got[:n], ref) and np.all(got[n:] == 0xEE), n
        dq = bk.cpu().numpy().view(np.uint16)
        assert np.array_equal(dq[:n], orc.fp8_dequantize(ref, sc)) and np.all(dq[n:] == 0x7777), n


def test_fp8_capsule_restore_then_lazy_stage_rebuild(orc):
    """Live set with FP8 K/V regions (one byte per element) and a recurrent
    state: the capsule holds half the K/V bytes of bf16; after a restore into
    a poisoned set the BF16 stage rebuilt from the FP8 rows equals the cold
    path's stage bit for bit."""
    import torch
    rows, heads, d, P, C = 512, 4, 64, 320, 64
    row_el = heads * d
    scale = 0.125
    rng = np.random.default_rng(7)
    kv_bf16 = [torch.from_numpy((rng.standard_normal((rows, row_el)) * 0.5).astype(np.float32)).to(torch.bfloat16).cuda()
               for _ in range(2)]
    fp8 = [torch.zeros(rows * row_el, dtype=torch.uint8, device="cuda") for _ in range(2)]
    stage = [torch.zeros(rows * row_el, dtype=torch.int16, device="cuda") for _ in range(2)]
    state = device_bytes(2 * 64 * 64 * 4, seed=3, name="state")
    # the prefill writes rows [0, P) into the FP8 regions; the stage is built from them
    cap.kv_fp8_quantize([(kv_bf16[i], fp8[i], P * row_el, scale) for i in range(2)])
    cap.kv_fp8_dequantize([(fp8[i], stage[i], P * row_el, scale) for i in range(2)])
    torch.cuda.synchronize()
    cold_stage = [s[: P * row_el].clone() for s in stage]
    bufs = [("k", fp8[0], row_el, rows, cap.CAP_KIND_POSITIONAL), ("state", state, state.numel(), 1, cap.CAP_KIND_FIXED),
            ("v", fp8[1], row_el, rows, cap.CAP_KIND_POSITIONAL)]
    live = cap.cap_set_create(bufs, C, 9)
    cap.cap_set_set_position(live, P)
    nbytes = cap.capsule_bytes(live, P)
    assert nbytes == 2 * P * row_el + state.numel()  # one byte per K/V element
    arena = device_bytes(nbytes)
    c = cap.capsule_snapshot(live, P, 1, arena)
    fp8_before = [f.cpu().numpy() for f in fp8]
    state_before = state.cpu().numpy()
    for t in fp8 + [state]:
        t.fill_(0x3C)
    for s in stage:
        s.fill_(0x1234)
    assert cap.capsule_restore(c, live, 1) == P
    # the stage of the restored session is valid over no rows: rebuild [0, P')
    cap.kv_fp8_dequantize([(fp8[i], stage[i], P * row_el, scale) for i in range(2)])
    torch.cuda.synchronize()
    for i in range(2):
        assert np.array_equal(fp8[i].cpu().numpy()[: P * row_el], fp8_before[i][: P * row_el])
        assert torch.equal(stage[i][: P * row_el], cold_stage[i])
        want = orc.fp8_dequantize(fp8_before[i][: P * row_el], scale)
        assert np.array_equal(stage[i][: P * row_el].cpu().numpy().view(np.uint16), want)
    assert np.array_equal(state.cpu().numpy(), state_before)


def test_fp8_stage_valid_end_and_lazy_rebuild(orc):
    """The FP8 stage's valid end E through snapshot / restore / fork / append
    (§3 "Definition", cost model): the first read after each step converts
    exactly the rows the stage lacks, and the stage then equals the
    dequantisation of its FP8 rows bit for bit -- the oracle's, and the eager
    conversion of the same rows (the cold path's stage).  Restore converts
    nothing; in the set and lineage the capsule came from it keeps the rows
    recorded at the snapshot, elsewhere it drops to 0."""
    import torch
    rows, row_el, scale, C = 512, 128, 0.25, 64
    rng = np.random.default_rng(11)

    def bf16_rows(mult):
        x = (rng.standard_normal((rows, row_el)) * mult).astype(np.float32)
        return torch.from_numpy(x).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    A = [bf16_rows(0.7), bf16_rows(1.3)]        # K and V content of stream A
    B = [bf16_rows(0.5), bf16_rows(2.0)]        # another continuation
    codes = {"A": [orc.fp8_quantize(a, scale) for a in A], "B": [orc.fp8_quantize(b, scale) for b in B]}
    src = {k: [torch.from_numpy(c.reshape(-1).copy()).cuda() for c in v] for k, v in codes.items()}

    def make():
        fp8 = [torch.zeros(rows * row_el, dtype=torch.uint8, device="cuda") for _ in range(2)]
        stage = [torch.full((rows * row_el,), 0x7777, dtype=torch.int16, device="cuda") for _ in range(2)]
        state = device_bytes(64 * 64 * 4, seed=5, name="state")
        bufs = [("k", fp8[0], row_el, rows, cap.CAP_KIND_POSITIONAL), ("state", state, state.numel(), 1,
                                                                        cap.CAP_KIND_FIXED),
                ("v", fp8[1], row_el, rows, cap.CAP_KIND_POSITIONAL)]
        s = cap.cap_set_create(bufs, C, 3)
        cap.cap_set_bind_stage(s, 0, stage[0], scale)
        cap.cap_set_bind_stage(s, 2, stage[1], scale)
        return s, fp8, stage, state

    def append(s, stream, t0, t1):
        k, v = (src[stream][i][t0 * row_el:t1 * row_el] for i in range(2))
        assert k.numel() == v.numel() == (t1 - t0) * row_el   # the source rows exist (checked on the host)
        cap.cap_set_append(s, [k, None, v], t1 - t0)

    def check(s, fp8, stage, n, content):
        """rows [0, n) of each FP8 buffer and stage against content = [(stream, t0, t1), ...]."""
        torch.cuda.synchronize()
        for i in range(2):
            want_codes = np.concatenate([codes[k][i][t0:t1] for k, t0, t1 in content]).reshape(-1)
            assert np.array_equal(fp8[i][:n * row_el].cpu().numpy(), want_codes)
            got = stage[i][:n * row_el].cpu().numpy().view(np.uint16)
            assert np.array_equal(got, orc.fp8_dequantize(want_codes, scale))
            eager = torch.empty(n * row_el, dtype=torch.int16, device="cuda")
            cap.kv_fp8_dequantize([(fp8[i], eager, n * row_el, scale)])
            torch.cuda.synchronize()
            assert torch.equal(stage[i][:n * row_el], eager)
        assert cap.cap_stage_valid_end(s) >= n

    s, fp8, stage, state = make()
    append(s, "A", 0, 320)
    assert cap.cap_stage_acquire(s, 320) == 320
    check(s, fp8, stage, 320, [("A", 0, 320)])
    arena1 = device_bytes(cap.capsule_bytes(s, 320))
    c1 = cap.capsule_snapshot(s, 320, 1, arena1)
    assert cap.capsule_stage_end(c1) == 320
    append(s, "A", 320, 384)
    assert cap.cap_stage_acquire(s, 384) == 64
    # poison the FP8 rows and the state (the stage belongs to the session), restore
    for t in fp8 + [state]:
        t.fill_(0x5A)
    assert cap.capsule_restore(c1, s, 1) == 320
    assert cap.cap_stage_valid_end(s) == 320           # re-bound, nothing converted
    assert cap.cap_stage_acquire(s, 320) == 0
    check(s, fp8, stage, 320, [("A", 0, 320)])
    # continue along B from the boundary
    append(s, "B", 320, 384)
    assert cap.cap_stage_acquire(s, 384) == 64
    check(s, fp8, stage, 384, [("A", 0, 320), ("B", 320, 384)])
    arena2 = device_bytes(cap.capsule_bytes(s, 384))
    c2 = cap.capsule_snapshot(s, 384, 2, arena2)
    assert cap.capsule_stage_end(c2) == 384
    # c1 again: a restore happened since its snapshot, so the stage starts over
    assert cap.capsule_restore(c1, s, 1) == 320
    assert cap.cap_stage_valid_end(s) == 0
    assert cap.cap_stage_acquire(s, 320) == 320
    check(s, fp8, stage, 320, [("A", 0, 320)])
    assert cap.capsule_restore(c2, s, 2) == 384 and cap.cap_stage_valid_end(s) == 0
    assert cap.cap_stage_acquire(s, 200) == 200 and cap.cap_stage_acquire(s, 384) == 184
    check(s, fp8, stage, 384, [("A", 0, 320), ("B", 320, 384)])
    # another session: fork leaves its stage empty; its first read converts everything
    s2, fp8_2, stage_2, _ = make()
    cap.capsule_fork(c2, [s2], 2)
    assert cap.cap_stage_valid_end(s2) == 0 and cap.cap_stage_acquire(s2, 384) == 384
    check(s2, fp8_2, stage_2, 384, [("A", 0, 320), ("B", 320, 384)])
    # an append below rows the set already held clips E to the append position
    cap.cap_set_set_position(s, 352)
    append(s, "A", 352, 384)
    assert cap.cap_stage_valid_end(s) == 352
    assert cap.cap_stage_acquire(s, 384) == 32
    check(s, fp8, stage, 384, [("A", 0, 320), ("B", 320, 352), ("A", 352, 384)])
    # ... and that capsule c2 (taken before the rewrite) no longer matches the lineage
    assert cap.capsule_restore(c2, s, 2) == 384 and cap.cap_stage_valid_end(s) == 0
    # invalidation, errors
    cap.cap_stage_acquire(s, 384)
    cap.cap_stage_invalidate(s)
    assert cap.cap_stage_valid_end(s) == 0 and cap.cap_stage_acquire(s, 384) == 384
    for call, status in ((lambda: cap.cap_stage_acquire(s, 385), cap.CAP_E_SIZE),
                         (lambda: cap.cap_set_bind_stage(s, 1, stage[0], scale), cap.CAP_E_UNSUPPORTED),
                         (lambda: cap.cap_set_bind_stage(s, 0, fp8[1], scale), cap.CAP_E_INVAL),
                         (lambda: cap.cap_set_bind_stage(s, 0, stage_2[0], 0.0), cap.CAP_E_INVAL),
                         (lambda: cap.cap_set_bind_stage(s, 2, stage[0], scale), cap.CAP_E_INVAL)):
        with pytest.raises(cap.CapsuleError) as ei:
            call()
        assert ei.value.status == status
    plain = cap.cap_set_create([("x", device_bytes(4096), 64, 64, cap.CAP_KIND_POSITIONAL)], C, 1)
    with pytest.raises(cap.CapsuleError) as ei:
        cap.cap_stage_acquire(plain, 0)
    assert ei.value.status == cap.CAP_E_STATE
