"""The C-ABI library on the host, without a GPU: it loads, exports every
symbol include/capsule.h declares, and its host-side checks return the
documented status codes before any device call."""
import ctypes as ct
import os
import re

import numpy as np
import pytest

import paper_2606_20537_amd as cap
from paper_2606_20537_amd import _native as N

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "capsule.h")


def declared_symbols():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
    return sorted(set(re.findall(r"CAP_API\s+[\w\s\*]+?\b(\w+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    names = declared_symbols()
    assert len(names) >= 15, names
    lib = ct.CDLL(cap.build.LIB_PATH if hasattr(cap, "build") else N.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), "missing export %s" % n
    # the binding wraps exactly these entry points
    assert sorted(s[0] for s in N.SIGNATURES) == names


def test_status_strings():
    for code in (0, -1, -2, -3, -4, -5, -6, -7, -8):
        assert cap.cap_status_string(code) not in ("", "unknown status")
    assert cap.cap_status_string(-99) == "unknown status"


def test_align_matches_oracle(orc):
    rng = np.random.default_rng(0)
    for _ in range(2000):
        P = int(rng.integers(0, 1 << 40))
        C = int(rng.integers(1, 4096))
        assert cap.cap_align_boundary(P, C) == orc.align(P, C)
    assert cap.cap_align_boundary(123, 0) == 0


def test_digest_matches_oracle(orc):
    rng = np.random.default_rng(1)
    for n in (0, 1, 7, 2048):
        ids = rng.integers(-2**31, 2**31 - 1, size=n, dtype=np.int64).astype(np.int32)
        assert cap.capsule_digest_tokens(ids) == orc.digest_tokens(ids)


def _bufs(layout):
    return [(name, 0, rb, rows, kind) for name, rb, rows, kind in layout]


def test_layout_bytes_match_oracle(orc):
    rng = np.random.default_rng(2)
    for trial in range(200):
        n = int(rng.integers(1, 12))
        layout = []
        for i in range(n):
            kind = int(rng.integers(0, 2))
            layout.append(("b%d" % i, int(rng.integers(1, 64)) * 16, int(rng.integers(1, 300)), kind))
        chunk = int(rng.integers(1, 100))
        cap_rows = min([l[2] for l in layout if l[3] == 0], default=10**9)
        P = int(rng.integers(0, cap_rows + 1))
        got = cap.capsule_layout_bytes(_bufs(layout), chunk, P)
        want = orc.capsule_bytes([l[1] for l in layout], [l[2] for l in layout], [l[3] for l in layout],
                                 orc.align(P, chunk))
        assert got == want


def _status(fn, *a, **k):
    try:
        fn(*a, **k)
    except cap.CapsuleError as e:
        return e.status
    return cap.CAP_OK


def test_layout_errors():
    ok = [("k", 64, 100, 0), ("s", 256, 1, 1)]
    assert _status(cap.capsule_layout_bytes, _bufs(ok), 64, 64) == cap.CAP_OK
    assert _status(cap.capsule_layout_bytes, _bufs([("k", 64, 100, 7)]), 64, 0) == cap.CAP_E_UNSUPPORTED
    assert _status(cap.capsule_layout_bytes, _bufs([("k", 24, 100, 0)]), 64, 0) == cap.CAP_E_ALIGN
    assert _status(cap.capsule_layout_bytes, _bufs([("k", 64, 0, 0)]), 64, 0) == cap.CAP_E_INVAL
    assert _status(cap.capsule_layout_bytes, _bufs([("k", 64, 10, 0), ("k", 64, 10, 0)]), 64, 0) == cap.CAP_E_INVAL
    assert _status(cap.capsule_layout_bytes, _bufs(ok), 0, 0) == cap.CAP_E_INVAL
    assert _status(cap.capsule_layout_bytes, _bufs(ok), 64, 128) == cap.CAP_E_SIZE  # P' = 128 > 100 rows
    many = [("b%d" % i, 16, 1, 1) for i in range(cap.CAP_MAX_BUFFERS + 1)]
    assert _status(cap.capsule_layout_bytes, _bufs(many), 1, 0) == cap.CAP_E_UNSUPPORTED
    # sizes that fit 64 bits one by one but not in sum
    half = [("a", 1 << 62, 2, 1), ("b", 1 << 62, 2, 1)]
    assert _status(cap.capsule_layout_bytes, _bufs(half), 64, 0) == cap.CAP_E_SIZE
    assert _status(cap.capsule_layout_bytes, _bufs(half[:1]), 64, 0) == cap.CAP_OK


def test_set_create_rejects_before_device():
    # checks that run before the device table is built
    assert _status(cap.cap_set_create, [("k", 0, 64, 10, 0)], 64, 1) == cap.CAP_E_INVAL      # null pointer
    assert _status(cap.cap_set_create, [("k", 8, 64, 10, 0)], 64, 1) == cap.CAP_E_ALIGN      # misaligned
    assert _status(cap.cap_set_create, [("k", 4096, 64, 10, 3)], 64, 1) == cap.CAP_E_UNSUPPORTED
    overlapping = [("a", 4096, 64, 10, 0), ("b", 4096 + 320, 64, 10, 0)]
    assert _status(cap.cap_set_create, overlapping, 64, 1) == cap.CAP_E_INVAL
    # an address range that wraps past 2^64
    assert _status(cap.cap_set_create, [("k", (1 << 64) - 4096, 64, 100, 0)], 64, 1) == cap.CAP_E_SIZE


def test_null_handles():
    L = N.load()
    out = ct.c_uint64(0)
    assert L.capsule_bytes(None, 0, ct.byref(out)) == cap.CAP_E_INVAL
    assert L.cap_set_set_position(None, 0) == cap.CAP_E_INVAL
    assert L.cap_set_destroy(None) == cap.CAP_E_INVAL
    assert L.capsule_release(None) == cap.CAP_E_INVAL
    assert L.capsule_restore(None, None, 0, None, None) == cap.CAP_E_INVAL
    h = ct.c_void_p(1)
    assert L.capsule_snapshot(None, 0, 0, None, 0, None, ct.byref(h)) == cap.CAP_E_INVAL
    assert h.value is None  # *out cleared on error
    assert L.capsule_fork(None, None, 0, 0, None) == cap.CAP_E_INVAL
    assert L.capsule_gather_restore(None, 0, None, None, 0, None) == cap.CAP_E_INVAL
    assert L.linattn_chunked_prefill(None, None) == cap.CAP_E_INVAL
    assert L.linattn_decode_step(None, None) == cap.CAP_E_INVAL
    assert L.gdn_decode_step(None, None) == cap.CAP_E_INVAL
    h = ct.c_void_p(1)
    assert L.capsule_move(None, None, 0, None, ct.byref(h)) == cap.CAP_E_INVAL
    assert h.value is None
    assert L.capsule_move(None, None, 0, None, None) == cap.CAP_E_INVAL
    t = ct.c_uint32(9)
    assert L.capsule_tier(None, ct.byref(t)) == cap.CAP_E_INVAL and t.value == 9
    e = ct.c_uint64(0)
    assert L.cap_set_bind_stage(None, 0, None, ct.c_float(1.0)) == cap.CAP_E_INVAL
    assert L.cap_stage_acquire(None, 0, None, None) == cap.CAP_E_INVAL
    assert L.cap_stage_valid_end(None, ct.byref(e)) == cap.CAP_E_INVAL
    assert L.cap_stage_invalidate(None) == cap.CAP_E_INVAL
    assert L.capsule_stage_end(None, ct.byref(e)) == cap.CAP_E_INVAL


def _args(**kw):
    base = dict(q=4096, k=8192, v=12288, g=16384, state_in=0, o=1 << 30, chunk_states=0, final_state=0,
                T=4, H=1, dk=64, dv=16, chunk=64, in_dtype=cap.CAP_DTYPE_BF16, scale=1.0)
    base.update(kw)
    return N.linattn_args(**base)


def _scan_status(**kw):
    return N.load().linattn_chunked_prefill(ct.byref(_args(**kw)), None)


def test_scan_argument_checks():
    # every case below fails on the host before any launch
    assert _scan_status(T=-1) == cap.CAP_E_INVAL
    assert _scan_status(H=0) == cap.CAP_E_INVAL
    assert _scan_status(in_dtype=7) == cap.CAP_E_INVAL
    assert _scan_status(q=0) == cap.CAP_E_INVAL
    assert _scan_status(o=0) == cap.CAP_E_INVAL
    assert _scan_status(chunk=32) == cap.CAP_E_UNSUPPORTED
    assert _scan_status(dk=96) == cap.CAP_E_UNSUPPORTED
    assert _scan_status(dv=24) == cap.CAP_E_UNSUPPORTED
    assert _scan_status(dk=128, in_dtype=cap.CAP_DTYPE_F32) == cap.CAP_E_UNSUPPORTED
    assert _scan_status(q=4100) == cap.CAP_E_ALIGN
    assert _scan_status(final_state=4104) == cap.CAP_E_ALIGN
    # an output overlapping an input
    assert _scan_status(o=8192 + 64) == cap.CAP_E_INVAL
    # outputs overlapping each other
    assert _scan_status(final_state=1 << 30) == cap.CAP_E_INVAL
    # nothing to do: T = 0 without a final state returns at once
    assert _scan_status(T=0, q=0, k=0, v=0, g=0, o=0) == cap.CAP_OK
    # more heads than 32-bit offsets inside one state of all heads can address
    assert _scan_status(H=32768, dk=128, dv=128) == cap.CAP_E_UNSUPPORTED
    assert _scan_status(H=32767, dk=128, dv=128, T=0, q=0, k=0, v=0, g=0, o=0) == cap.CAP_OK
    # more chunks than the kernels count in 32 bits
    assert _scan_status(T=(1 << 36) + 1) == cap.CAP_E_UNSUPPORTED


def test_decode_step_argument_checks():
    """The decode step runs the prefill's checks, then requires T == 1."""
    L = N.load()
    for T in (0, 2, 64):
        assert L.linattn_decode_step(ct.byref(_args(T=T)), None) == cap.CAP_E_UNSUPPORTED
    assert L.linattn_decode_step(ct.byref(_args(T=1, q=0)), None) == cap.CAP_E_INVAL
    assert L.linattn_decode_step(ct.byref(_args(T=1, dk=96)), None) == cap.CAP_E_UNSUPPORTED
    assert L.linattn_decode_step(ct.byref(_args(T=1, o=8192 + 64)), None) == cap.CAP_E_INVAL
    g = dict(q=4096, k=8192, v=12288, g=16384, beta=20480, state_in=0, o=1 << 30, chunk_states=0,
             final_state=0, workspace=0, workspace_bytes=0, T=2, H=1, dk=64, dv=16, chunk=64,
             in_dtype=cap.CAP_DTYPE_BF16, scale=1.0)
    assert L.gdn_decode_step(ct.byref(N.gdn_args(**g)), None) == cap.CAP_E_UNSUPPORTED
    g.update(T=1, beta=0)
    assert L.gdn_decode_step(ct.byref(N.gdn_args(**g)), None) == cap.CAP_E_INVAL
    g.update(beta=20484)
    assert L.gdn_decode_step(ct.byref(N.gdn_args(**g)), None) == cap.CAP_E_ALIGN


OOM_DRIVER = r"""
#include <cstdio>
#include <cstdlib>
#include <new>
#include "capsule.h"
// Global operator new of this executable interposes the library's: once
// g_fail is set, every host allocation fails.
static bool g_fail = false;
void* operator new(std::size_t n) {
    if (g_fail) throw std::bad_alloc();
    void* p = std::malloc(n ? n : 1);
    if (!p) throw std::bad_alloc();
    return p;
}
void* operator new(std::size_t n, const std::nothrow_t&) noexcept { return g_fail ? nullptr : std::malloc(n ? n : 1); }
void operator delete(void* p) noexcept { std::free(p); }
void operator delete(void* p, std::size_t) noexcept { std::free(p); }
int main() {
    cap_buf b[2] = {{"k", (void*)4096, 64, 10, CAP_KIND_POSITIONAL, 0}, {"s", (void*)65536, 256, 1, CAP_KIND_FIXED, 0}};
    uint64_t bytes = 0;
    const int ok = capsule_layout_bytes(b, 2, 64, 0, &bytes);
    g_fail = true;
    const int oom_layout = capsule_layout_bytes(b, 2, 64, 0, &bytes);
    cap_set s = (cap_set)1;
    const int oom_create = cap_set_create(b, 2, 64, 1, &s);
    g_fail = false;
    std::printf("%d %d %d %d\n", ok, oom_layout, oom_create, s == nullptr);
    return 0;
}
"""


def test_host_allocation_failure_is_nomem(tmp_path):
    """A host allocation that fails inside an entry point returns CAP_E_NOMEM
    (no exception crosses the C boundary) and leaves *out cleared; checked
    with a driver whose operator new fails on demand."""
    import shutil
    import subprocess
    if shutil.which("g++") is None:
        pytest.skip("g++ not available")
    libdir = os.path.dirname(N.LIB_PATH)
    src = tmp_path / "oom.cpp"
    src.write_text(OOM_DRIVER)
    exe = tmp_path / "oom"
    subprocess.run(["g++", "-std=c++17", "-O1", "-I", os.path.join(ROOT, "include"), "-o", str(exe), str(src),
                    "-L" + libdir, "-lcapsule", "-Wl,-rpath," + libdir, "-Wl,-rpath,/opt/rocm/lib"], check=True)
    out = subprocess.run([str(exe)], check=True, capture_output=True, text=True).stdout.split()
    assert out == [str(cap.CAP_OK), str(cap.CAP_E_NOMEM), str(cap.CAP_E_NOMEM), "1"], out


def _gdn_status(**kw):
    base = dict(q=4096, k=8192, v=12288, g=16384, beta=20480, state_in=0, o=1 << 30, chunk_states=0,
                final_state=0, workspace=1 << 31, workspace_bytes=12800, T=4, H=1, dk=64, dv=16, chunk=64,
                in_dtype=cap.CAP_DTYPE_BF16, scale=1.0)
    base.update(kw)
    return N.load().gdn_chunked_prefill(ct.byref(N.gdn_args(**base)), None)


def test_gdn_argument_checks():
    L = N.load()
    assert L.gdn_chunked_prefill(None, None) == cap.CAP_E_INVAL
    assert L.gdn_workspace_bytes(0, 4, 64) == 0 and L.gdn_workspace_bytes(65, 3, 64) == 2 * 3 * 12800
    assert L.gdn_workspace_bytes(65, 3, 32) == 0
    assert _gdn_status(T=-1) == cap.CAP_E_INVAL
    assert _gdn_status(H=0) == cap.CAP_E_INVAL
    assert _gdn_status(in_dtype=7) == cap.CAP_E_INVAL
    assert _gdn_status(in_dtype=cap.CAP_DTYPE_F32) == cap.CAP_E_UNSUPPORTED
    for name in ("q", "k", "v", "g", "beta", "o", "workspace"):
        assert _gdn_status(**{name: 0}) == cap.CAP_E_INVAL, name
    assert _gdn_status(chunk=32) == cap.CAP_E_UNSUPPORTED
    assert _gdn_status(dk=96) == cap.CAP_E_UNSUPPORTED
    assert _gdn_status(dv=24) == cap.CAP_E_UNSUPPORTED
    assert _gdn_status(workspace_bytes=12800 - 16) == cap.CAP_E_SIZE
    assert _gdn_status(beta=20484) == cap.CAP_E_ALIGN
    assert _gdn_status(workspace=(1 << 31) + 8) == cap.CAP_E_ALIGN
    # the workspace overlapping an input, an output overlapping the workspace
    assert _gdn_status(workspace=20480) == cap.CAP_E_INVAL
    assert _gdn_status(o=(1 << 31) + 4096) == cap.CAP_E_INVAL
    assert _gdn_status(o=12288 + 32) == cap.CAP_E_INVAL
    # nothing to do: T = 0 without a final state returns at once, no workspace needed
    assert _gdn_status(T=0, q=0, k=0, v=0, g=0, beta=0, o=0, workspace=0, workspace_bytes=0) == cap.CAP_OK
    # more heads than 32-bit offsets inside one state of all heads can address
    assert _gdn_status(H=32768, dk=128, dv=128) == cap.CAP_E_UNSUPPORTED


def test_python_binding_has_no_fallback(tmp_path):
    with pytest.raises(ImportError):
        N.load(str(tmp_path / "missing.so"))


def _fp8_status(segs, quantize=True):
    arr = (N.kv_fp8_seg * max(1, len(segs)))()
    for i, (src, dst, n, scale, res) in enumerate(segs):
        arr[i] = N.kv_fp8_seg(src, dst, n, scale, res)
    fn = N.load().kv_fp8_quantize if quantize else N.load().kv_fp8_dequantize
    return fn(arr, len(segs), None)


def test_fp8_argument_checks():
    ok = (1 << 20, 1 << 24, 1024, 1.0, 0)
    for q in (True, False):
        assert N.load().kv_fp8_quantize(None, 1, None) == cap.CAP_E_INVAL
        assert _fp8_status([], q) == cap.CAP_E_INVAL
        assert _fp8_status([ok] * 65, q) == cap.CAP_E_UNSUPPORTED
        assert _fp8_status([(1 << 20, 1 << 24, 1000, 1.0, 0)], q) == cap.CAP_E_ALIGN     # n % 16
        assert _fp8_status([((1 << 20) + 8, 1 << 24, 1024, 1.0, 0)], q) == cap.CAP_E_ALIGN
        assert _fp8_status([(1 << 20, 1 << 24, 1024, 0.0, 0)], q) == cap.CAP_E_INVAL
        assert _fp8_status([(1 << 20, 1 << 24, 1024, -1.0, 0)], q) == cap.CAP_E_INVAL
        assert _fp8_status([(1 << 20, 1 << 24, 1024, float("nan"), 0)], q) == cap.CAP_E_INVAL
        assert _fp8_status([(1 << 20, 1 << 24, 1024, float("inf"), 0)], q) == cap.CAP_E_INVAL
        assert _fp8_status([(1 << 20, 1 << 24, 1024, 1.0, 1)], q) == cap.CAP_E_INVAL
        assert _fp8_status([(0, 1 << 24, 1024, 1.0, 0)], q) == cap.CAP_E_INVAL
        assert _fp8_status([(1 << 20, (1 << 20) + 512, 1024, 1.0, 0)], q) == cap.CAP_E_INVAL   # src/dst overlap
        two = [(1 << 20, 1 << 24, 1024, 1.0, 0), (1 << 21, (1 << 24) + 512, 1024, 1.0, 0)]
        assert _fp8_status(two, q) == cap.CAP_E_INVAL                                        # dst overlap



def test_noalloc_argument_checks():
    """The no-allocation delta-rule prefill: the prefill's checks, no
    workspace argument, and CAP_E_SIZE when one chunk of all heads does not
    fit its fixed scratch -- all on the host before any device call."""
    L = N.load()
    assert L.gdn_chunked_prefill_noalloc(None, None) == cap.CAP_E_INVAL
    base = dict(q=4096, k=8192, v=12288, g=16384, beta=20480, state_in=0, o=1 << 30, chunk_states=0,
                final_state=0, workspace=0, workspace_bytes=0, T=4, H=1, dk=64, dv=16, chunk=64,
                in_dtype=cap.CAP_DTYPE_BF16, scale=1.0)

    def st(**kw):
        a = dict(base)
        a.update(kw)
        return L.gdn_chunked_prefill_noalloc(ct.byref(N.gdn_args(**a)), None)
    assert st(workspace=1 << 31, workspace_bytes=12800) == cap.CAP_E_INVAL
    assert st(workspace_bytes=16) == cap.CAP_E_INVAL
    assert st(beta=0) == cap.CAP_E_INVAL
    assert st(dk=96) == cap.CAP_E_UNSUPPORTED
    assert st(T=0, q=0, k=0, v=0, g=0, beta=0, o=0, H=300, dk=128, dv=128) == cap.CAP_E_SIZE
    assert st(T=0, q=0, k=0, v=0, g=0, beta=0, o=0, H=233, dk=128, dv=128) == cap.CAP_OK
    assert st(T=0, q=0, k=0, v=0, g=0, beta=0, o=0, H=234, dk=128, dv=128) == cap.CAP_E_SIZE
    assert cap.GDN_NOALLOC_SCRATCH_BYTES == 32 << 20
