"""ctypes binding of libcapsule.so: argument marshalling only.

Every function here has the name of the C entry point it calls (include/
capsule.h) and forwards to it; all work runs in the library's HIP kernels.
Device buffers are passed as torch tensors (their data pointers) or as raw
integer addresses; streams as torch streams, raw hipStream_t integers or
None (torch's current stream).  A non-zero status raises CapsuleError.
There is no fallback: if the library is missing, loading raises.
"""
import ctypes as ct
import os

from .build import LIB_PATH

CAP_OK = 0
CAP_E_INVAL = -1
CAP_E_SIZE = -2
CAP_E_DIGEST = -3
CAP_E_UNSUPPORTED = -4
CAP_E_ALIGN = -5
CAP_E_STATE = -6
CAP_E_HIP = -7
CAP_E_NOMEM = -8

CAP_KIND_POSITIONAL = 0
CAP_KIND_FIXED = 1
CAP_TIER_DEVICE = 0
CAP_TIER_HOST = 1
CAP_DTYPE_F32 = 0
CAP_DTYPE_BF16 = 1

CAP_MAX_BUFFERS = 512
CAP_MAX_FORK = 16
CAP_MAX_GALLERY = 64
CAP_MAX_STAGES = 64


class CapsuleError(RuntimeError):
    def __init__(self, fn, status, msg):
        super().__init__("%s failed: %d (%s)" % (fn, status, msg))
        self.status = status
        self.fn = fn


class cap_buf(ct.Structure):
    _fields_ = [("name", ct.c_char_p), ("dptr", ct.c_void_p), ("row_bytes", ct.c_uint64),
                ("rows", ct.c_uint64), ("kind", ct.c_uint32), ("reserved", ct.c_uint32)]


class linattn_args(ct.Structure):
    _fields_ = [("q", ct.c_void_p), ("k", ct.c_void_p), ("v", ct.c_void_p), ("g", ct.c_void_p),
                ("state_in", ct.c_void_p), ("o", ct.c_void_p), ("chunk_states", ct.c_void_p),
                ("final_state", ct.c_void_p), ("T", ct.c_int64), ("H", ct.c_int32), ("dk", ct.c_int32),
                ("dv", ct.c_int32), ("chunk", ct.c_int32), ("in_dtype", ct.c_int32), ("scale", ct.c_float)]


class gdn_args(ct.Structure):
    _fields_ = [("q", ct.c_void_p), ("k", ct.c_void_p), ("v", ct.c_void_p), ("g", ct.c_void_p),
                ("beta", ct.c_void_p), ("state_in", ct.c_void_p), ("o", ct.c_void_p),
                ("chunk_states", ct.c_void_p), ("final_state", ct.c_void_p), ("workspace", ct.c_void_p),
                ("workspace_bytes", ct.c_uint64), ("T", ct.c_int64), ("H", ct.c_int32), ("dk", ct.c_int32),
                ("dv", ct.c_int32), ("chunk", ct.c_int32), ("in_dtype", ct.c_int32), ("scale", ct.c_float)]


class kv_fp8_seg(ct.Structure):
    _fields_ = [("src", ct.c_void_p), ("dst", ct.c_void_p), ("n", ct.c_uint64), ("scale", ct.c_float),
                ("reserved", ct.c_uint32)]


# (name, restype, argtypes) of every exported entry point
_vp, _u64, _u32, _i32 = ct.c_void_p, ct.c_uint64, ct.c_uint32, ct.c_int32
SIGNATURES = [
    ("cap_status_string", ct.c_char_p, [ct.c_int]),
    ("cap_align_boundary", _u64, [_u64, _u32]),
    ("capsule_layout_bytes", ct.c_int, [ct.POINTER(cap_buf), _u32, _u32, _u64, ct.POINTER(_u64)]),
    ("cap_set_create", ct.c_int, [ct.POINTER(cap_buf), _u32, _u32, _u64, ct.POINTER(_vp)]),
    ("cap_set_destroy", ct.c_int, [_vp]),
    ("cap_set_set_position", ct.c_int, [_vp, _u64]),
    ("cap_set_get_position", ct.c_int, [_vp, ct.POINTER(_u64)]),
    ("cap_set_append", ct.c_int, [_vp, ct.POINTER(_vp), _u64, _vp]),
    ("capsule_bytes", ct.c_int, [_vp, _u64, ct.POINTER(_u64)]),
    ("capsule_snapshot", ct.c_int, [_vp, _u64, _u64, _vp, _u64, _vp, ct.POINTER(_vp)]),
    ("capsule_restore", ct.c_int, [_vp, _vp, _u64, _vp, ct.POINTER(_u64)]),
    ("capsule_fork", ct.c_int, [_vp, ct.POINTER(_vp), _u32, _u64, _vp]),
    ("capsule_gather_restore", ct.c_int, [ct.POINTER(_vp), _u32, ct.POINTER(_i32), ct.POINTER(_vp), _u32, _vp]),
    ("capsule_info", ct.c_int, [_vp, ct.POINTER(_u64), ct.POINTER(_u64), ct.POINTER(_u64), ct.POINTER(_u64),
                                ct.POINTER(_vp)]),
    ("capsule_move", ct.c_int, [_vp, _vp, _u64, _vp, ct.POINTER(_vp)]),
    ("kv_fp8_quantize", ct.c_int, [ct.POINTER(kv_fp8_seg), _u32, _vp]),
    ("kv_fp8_dequantize", ct.c_int, [ct.POINTER(kv_fp8_seg), _u32, _vp]),
    ("capsule_tier", ct.c_int, [_vp, ct.POINTER(_u32)]),
    ("cap_set_bind_stage", ct.c_int, [_vp, _u32, _vp, ct.c_float]),
    ("cap_stage_acquire", ct.c_int, [_vp, _u64, _vp, ct.POINTER(_u64)]),
    ("cap_stage_valid_end", ct.c_int, [_vp, ct.POINTER(_u64)]),
    ("cap_stage_invalidate", ct.c_int, [_vp]),
    ("capsule_stage_end", ct.c_int, [_vp, ct.POINTER(_u64)]),
    ("capsule_release", ct.c_int, [_vp]),
    ("capsule_digest_tokens", _u64, [ct.POINTER(_i32), _u64]),
    ("linattn_chunked_prefill", ct.c_int, [ct.POINTER(linattn_args), _vp]),
    ("linattn_decode_step", ct.c_int, [ct.POINTER(linattn_args), _vp]),
    ("gdn_workspace_bytes", _u64, [ct.c_int64, _i32, _i32]),
    ("gdn_chunked_prefill", ct.c_int, [ct.POINTER(gdn_args), _vp]),
    ("gdn_decode_step", ct.c_int, [ct.POINTER(gdn_args), _vp]),
    ("gdn_chunked_prefill_noalloc", ct.c_int, [ct.POINTER(gdn_args), _vp]),
]

_lib = None


def load(path: str = LIB_PATH):
    """Load libcapsule.so (built by ``paper_2606_20537_amd.build``)."""
    global _lib
    if _lib is not None and path == LIB_PATH:
        return _lib
    if not os.path.exists(path):
        raise ImportError("libcapsule.so is not built (%s); run paper_2606_20537_amd.build.build()" % path)
    lib = ct.CDLL(path)
    for name, res, args in SIGNATURES:
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    if path == LIB_PATH:
        _lib = lib
    return lib


def _check(fn, status):
    if status != CAP_OK:
        raise CapsuleError(fn, status, load().cap_status_string(status).decode())
    return status


def _addr(x):
    """Device address of a torch tensor or an int (None -> 0)."""
    if x is None:
        return 0
    if isinstance(x, int):
        return x
    return x.data_ptr()


def _stream(s):
    if s is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(s, int):
        return s
    return s.cuda_stream


class CapSet:
    """Handle of a live set (owns the C handle; destroy() or GC frees it).
    The set only points at its buffers, so the handle keeps the buffer
    objects (tensors) alive while it lives."""

    def __init__(self, handle, names, n, buffers=()):
        self.handle = handle
        self.names = names
        self.n = n
        self.buffers = list(buffers)

    def destroy(self):
        cap_set_destroy(self)

    def __del__(self):
        try:
            self.destroy()
        except Exception:
            pass


class Capsule:
    """Host header of one capsule; the arena is the caller's."""

    def __init__(self, handle, arena_ref):
        self.handle = handle
        self.arena_ref = arena_ref  # keeps a torch arena alive while the header lives

    def release(self):
        capsule_release(self)

    def __del__(self):
        try:
            self.release()
        except Exception:
            pass


def make_bufs(bufs):
    """bufs: iterable of (name, tensor_or_addr, row_bytes, rows, kind)."""
    bufs = list(bufs)
    arr = (cap_buf * len(bufs))()
    keep = []
    for i, (name, t, rb, rows, kind) in enumerate(bufs):
        nb = name.encode() if name is not None else None
        keep.append(nb)
        arr[i] = cap_buf(nb, _addr(t), int(rb), int(rows), int(kind), 0)
    return arr, keep


# ------------------------------------------------------------ entry points --
def cap_status_string(status):
    return load().cap_status_string(int(status)).decode()


def cap_align_boundary(P, chunk):
    return int(load().cap_align_boundary(int(P), int(chunk)))


def capsule_layout_bytes(bufs, chunk, P):
    arr, _keep = make_bufs(bufs)
    out = _u64(0)
    _check("capsule_layout_bytes", load().capsule_layout_bytes(arr, len(arr), int(chunk), int(P), ct.byref(out)))
    return int(out.value)


def cap_set_create(bufs, chunk, deploy_key):
    arr, keep = make_bufs(bufs)
    h = _vp()
    _check("cap_set_create", load().cap_set_create(arr, len(arr), int(chunk), int(deploy_key) & (2**64 - 1),
                                                    ct.byref(h)))
    return CapSet(h.value, [k.decode() if k else None for k in keep], len(arr),
                  [b[1] for b in bufs if not isinstance(b[1], int)])


def cap_set_destroy(s):
    """Free the set's C handle; the handle is cleared first, so a second
    destroy (explicit or by the garbage collector) is a no-op."""
    h, s.handle = s.handle, None
    if not h:
        return CAP_OK
    return _check("cap_set_destroy", load().cap_set_destroy(h))


def cap_set_set_position(s, position):
    return _check("cap_set_set_position", load().cap_set_set_position(s.handle, int(position)))


def cap_set_get_position(s):
    out = _u64(0)
    _check("cap_set_get_position", load().cap_set_get_position(s.handle, ct.byref(out)))
    return int(out.value)


def cap_set_append(s, srcs, n, stream=None):
    """Append n tokens: srcs has one entry per buffer of the set (tensor,
    address or None)."""
    if len(srcs) != s.n:
        raise ValueError("cap_set_append: %d sources for a set of %d buffers" % (len(srcs), s.n))
    arr = (_vp * len(srcs))(*[None if x is None else _addr(x) for x in srcs])
    return _check("cap_set_append", load().cap_set_append(s.handle, arr, int(n), _stream(stream)))


def capsule_bytes(s, P):
    out = _u64(0)
    _check("capsule_bytes", load().capsule_bytes(s.handle, int(P), ct.byref(out)))
    return int(out.value)


def capsule_snapshot(s, P, prefix_digest, arena, arena_bytes=None, stream=None):
    if arena_bytes is None:
        arena_bytes = arena.numel() * arena.element_size()
    h = _vp()
    _check("capsule_snapshot", load().capsule_snapshot(s.handle, int(P), int(prefix_digest) & (2**64 - 1),
                                                        _addr(arena), int(arena_bytes), _stream(stream),
                                                        ct.byref(h)))
    return Capsule(h.value, arena)


def capsule_restore(cap, s, prefix_digest, stream=None):
    out = _u64(0)
    _check("capsule_restore", load().capsule_restore(cap.handle, s.handle, int(prefix_digest) & (2**64 - 1),
                                                      _stream(stream), ct.byref(out)))
    return int(out.value)


def capsule_fork(cap, sets, prefix_digest, stream=None):
    arr = (_vp * len(sets))(*[s.handle for s in sets])
    return _check("capsule_fork", load().capsule_fork(cap.handle, arr, len(sets), int(prefix_digest) & (2**64 - 1),
                                                      _stream(stream)))


def capsule_gather_restore(gallery, ids, sets, stream=None):
    gal = (_vp * len(gallery))(*[c.handle for c in gallery])
    ids_arr = (_i32 * len(ids))(*[int(i) for i in ids])
    arr = (_vp * len(sets))(*[s.handle for s in sets])
    return _check("capsule_gather_restore", load().capsule_gather_restore(gal, len(gallery), ids_arr, arr,
                                                                          len(sets), _stream(stream)))


def capsule_info(cap):
    P, nb, pd, dk, ar = _u64(0), _u64(0), _u64(0), _u64(0), _vp()
    _check("capsule_info", load().capsule_info(cap.handle, ct.byref(P), ct.byref(nb), ct.byref(pd), ct.byref(dk),
                                               ct.byref(ar)))
    return {"P_aligned": int(P.value), "bytes": int(nb.value), "prefix_digest": int(pd.value),
            "deploy_key": int(dk.value), "arena": int(ar.value or 0)}


def capsule_move(cap, arena, arena_bytes=None, stream=None):
    """Copy a capsule into another arena (device memory, or a pinned host tensor)
    and return a capsule over it: device -> host demotes, host -> device promotes."""
    if arena_bytes is None:
        arena_bytes = arena.numel() * arena.element_size()
    h = _vp()
    _check("capsule_move", load().capsule_move(cap.handle, _addr(arena), int(arena_bytes), _stream(stream),
                                                ct.byref(h)))
    return Capsule(h.value, arena)


def capsule_tier(cap):
    out = _u32(0)
    _check("capsule_tier", load().capsule_tier(cap.handle, ct.byref(out)))
    return int(out.value)


def cap_set_bind_stage(s, buffer, stage, scale):
    """Bind FP8 positional buffer ``buffer`` (index in the set) to a bf16
    working stage (tensor or address) decoded with ``scale``."""
    return _check("cap_set_bind_stage", load().cap_set_bind_stage(s.handle, int(buffer), _addr(stage), float(scale)))


def cap_stage_acquire(s, rows, stream=None):
    """Make rows [0, rows) of the set's stages valid; returns the rows converted."""
    out = _u64(0)
    _check("cap_stage_acquire", load().cap_stage_acquire(s.handle, int(rows), _stream(stream), ct.byref(out)))
    return int(out.value)


def cap_stage_valid_end(s):
    out = _u64(0)
    _check("cap_stage_valid_end", load().cap_stage_valid_end(s.handle, ct.byref(out)))
    return int(out.value)


def cap_stage_invalidate(s):
    return _check("cap_stage_invalidate", load().cap_stage_invalidate(s.handle))


def capsule_stage_end(cap):
    out = _u64(0)
    _check("capsule_stage_end", load().capsule_stage_end(cap.handle, ct.byref(out)))
    return int(out.value)


def capsule_release(cap):
    """Free the capsule's host header; the handle is cleared first, so a
    second release (explicit or by the garbage collector) is a no-op."""
    h, cap.handle = cap.handle, None
    if not h:
        return CAP_OK
    return _check("capsule_release", load().capsule_release(h))


def capsule_digest_tokens(ids):
    import numpy as np
    a = np.ascontiguousarray(ids, dtype=np.int32)
    return int(load().capsule_digest_tokens(a.ctypes.data_as(ct.POINTER(_i32)), a.size))


def _linattn_args(q, k, v, g, o, state_in, chunk_states, final_state, T, H, dk, dv, chunk, in_dtype, scale):
    if T is None:
        T, H, dk = q.shape
        dv = v.shape[2]
    if in_dtype is None:
        import torch
        in_dtype = CAP_DTYPE_F32 if q.dtype == torch.float32 else CAP_DTYPE_BF16
    return linattn_args(_addr(q), _addr(k), _addr(v), _addr(g), _addr(state_in), _addr(o), _addr(chunk_states),
                        _addr(final_state), int(T), int(H), int(dk), int(dv), int(chunk), int(in_dtype),
                        float(scale))


def linattn_chunked_prefill(q, k, v, g, o, *, state_in=None, chunk_states=None, final_state=None,
                            T=None, H=None, dk=None, dv=None, chunk=64, in_dtype=None, scale=1.0,
                            stream=None):
    """Marshal tensors (or addresses with explicit sizes) into linattn_args."""
    a = _linattn_args(q, k, v, g, o, state_in, chunk_states, final_state, T, H, dk, dv, chunk, in_dtype, scale)
    return _check("linattn_chunked_prefill", load().linattn_chunked_prefill(ct.byref(a), _stream(stream)))


def linattn_decode_step(q, k, v, g, o, *, state_in=None, final_state=None, T=None, H=None, dk=None, dv=None,
                        chunk=64, in_dtype=None, scale=1.0, stream=None):
    """One decode token (T == 1): the same arguments as linattn_chunked_prefill."""
    a = _linattn_args(q, k, v, g, o, state_in, None, final_state, T, H, dk, dv, chunk, in_dtype, scale)
    return _check("linattn_decode_step", load().linattn_decode_step(ct.byref(a), _stream(stream)))


def gdn_workspace_bytes(T, H, chunk=64):
    """Bytes of device workspace gdn_chunked_prefill needs for T tokens, H heads."""
    return int(load().gdn_workspace_bytes(int(T), int(H), int(chunk)))


def gdn_chunked_prefill(q, k, v, g, beta, o, *, state_in=None, chunk_states=None, final_state=None,
                        workspace=None, workspace_bytes=None, T=None, H=None, dk=None, dv=None, chunk=64,
                        in_dtype=CAP_DTYPE_BF16, scale=1.0, stream=None):
    """Marshal tensors (or addresses with explicit sizes) into gdn_args.

    With no workspace given, one is allocated as a torch uint8 tensor on q's
    device for the duration of the call (stream-ordered by torch's caching
    allocator)."""
    if T is None:
        T, H, dk = q.shape
        dv = v.shape[2]
    need = gdn_workspace_bytes(T, H, chunk) if chunk > 0 and H > 0 else 0
    if workspace is None and need > 0:
        import torch
        workspace = torch.empty(need, dtype=torch.uint8, device=q.device)
    if workspace_bytes is None:
        workspace_bytes = workspace.numel() * workspace.element_size() if hasattr(workspace, "numel") else need
    a = gdn_args(_addr(q), _addr(k), _addr(v), _addr(g), _addr(beta), _addr(state_in), _addr(o),
                 _addr(chunk_states), _addr(final_state), _addr(workspace), int(workspace_bytes), int(T), int(H),
                 int(dk), int(dv), int(chunk), int(in_dtype), float(scale))
    return _check("gdn_chunked_prefill", load().gdn_chunked_prefill(ct.byref(a), _stream(stream)))


GDN_NOALLOC_SCRATCH_BYTES = 32 << 20


def gdn_chunked_prefill_noalloc(q, k, v, g, beta, o, *, state_in=None, chunk_states=None, final_state=None,
                                T=None, H=None, dk=None, dv=None, chunk=64, in_dtype=CAP_DTYPE_BF16, scale=1.0,
                                stream=None):
    """gdn_chunked_prefill with the library's own device scratch: no
    workspace argument, nothing allocated."""
    if T is None:
        T, H, dk = q.shape
        dv = v.shape[2]
    a = gdn_args(_addr(q), _addr(k), _addr(v), _addr(g), _addr(beta), _addr(state_in), _addr(o),
                 _addr(chunk_states), _addr(final_state), 0, 0, int(T), int(H), int(dk), int(dv), int(chunk),
                 int(in_dtype), float(scale))
    return _check("gdn_chunked_prefill_noalloc", load().gdn_chunked_prefill_noalloc(ct.byref(a), _stream(stream)))


def gdn_decode_step(q, k, v, g, beta, o, *, state_in=None, final_state=None, T=None, H=None, dk=None, dv=None,
                    chunk=64, in_dtype=CAP_DTYPE_BF16, scale=1.0, stream=None):
    """One decode token (T == 1) of the delta rule; no workspace."""
    if T is None:
        T, H, dk = q.shape
        dv = v.shape[2]
    a = gdn_args(_addr(q), _addr(k), _addr(v), _addr(g), _addr(beta), _addr(state_in), _addr(o), 0,
                 _addr(final_state), 0, 0, int(T), int(H), int(dk), int(dv), int(chunk), int(in_dtype),
                 float(scale))
    return _check("gdn_decode_step", load().gdn_decode_step(ct.byref(a), _stream(stream)))


def _fp8_segs(segs):
    """segs: iterable of (src, dst, n_elements, scale); src/dst tensors or addresses."""
    segs = list(segs)
    arr = (kv_fp8_seg * max(1, len(segs)))()
    for i, (src, dst, n, scale) in enumerate(segs):
        arr[i] = kv_fp8_seg(_addr(src), _addr(dst), int(n), float(scale), 0)
    return arr, len(segs)


def kv_fp8_quantize(segs, stream=None):
    """bf16 -> OCP E4M3 for each (src, dst, n, scale) segment, one launch."""
    arr, n = _fp8_segs(segs)
    return _check("kv_fp8_quantize", load().kv_fp8_quantize(arr, n, _stream(stream)))


def kv_fp8_dequantize(segs, stream=None):
    """OCP E4M3 -> bf16 for each (src, dst, n, scale) segment, one launch."""
    arr, n = _fp8_segs(segs)
    return _check("kv_fp8_dequantize", load().kv_fp8_dequantize(arr, n, _stream(stream)))
