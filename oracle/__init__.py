"""CPU oracle for the capsule + chunked-scan hot path -- TEST INFRASTRUCTURE.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  The product library and its Python
binding never import it, and it never imports them.

The arithmetic lives in plain C (``linattn_oracle.c``, ``capsule_oracle.c``,
fp64 accumulation); this module only marshals numpy arrays through ctypes.
Each wrapper names the passage of the paper ("Execution-State Capsules") that
the underlying C function follows.
"""
import ctypes as ct
import os

import numpy as np

from . import build as _build

KIND_POSITIONAL = 0
KIND_FIXED = 1

_f32p = np.ctypeslib.ndpointer(dtype=np.float32, flags="C_CONTIGUOUS")
_f64p = np.ctypeslib.ndpointer(dtype=np.float64, flags="C_CONTIGUOUS")


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ct.c_void_p)


class Oracle:
    """Handle on one build of the oracle library (the default build, or a
    deliberately modified copy used by the mutation tests)."""

    def __init__(self, lib_path: str):
        self.path = lib_path
        L = ct.CDLL(lib_path)
        vp, i64, u64, u32 = ct.c_void_p, ct.c_int64, ct.c_uint64, ct.c_uint32
        L.orc_linattn_sequential.argtypes = [i64, i64, i64, i64, vp, vp, vp, vp, ct.c_double, vp, vp, vp]
        L.orc_linattn_sequential.restype = ct.c_int
        L.orc_linattn_chunked.argtypes = [i64, i64, i64, i64, i64, vp, vp, vp, vp, ct.c_double, vp, vp, vp, vp]
        L.orc_linattn_chunked.restype = ct.c_int
        L.orc_align.argtypes = [u64, u64]
        L.orc_align.restype = u64
        L.orc_capsule_bytes.argtypes = [u32, vp, vp, vp, u64]
        L.orc_capsule_bytes.restype = u64
        L.orc_capsule_snapshot.argtypes = [u32, vp, vp, vp, vp, u64, vp]
        L.orc_capsule_restore.argtypes = [u32, vp, vp, vp, vp, u64, vp]
        L.orc_capsule_fork.argtypes = [u32, u32, vp, vp, vp, vp, u64, vp]
        L.orc_capsule_gather.argtypes = [u32, u32, vp, vp, vp, vp, u64, u32, vp, vp]
        L.orc_capsule_gather.restype = ct.c_int
        L.orc_set_append.argtypes = [u32, vp, vp, vp, vp, vp, u64, u64, vp]
        L.orc_set_append.restype = ct.c_int
        L.orc_digest_tokens.argtypes = [vp, u64]
        L.orc_digest_tokens.restype = u64
        L.orc_digest_bytes.argtypes = [vp, u64]
        L.orc_digest_bytes.restype = u64
        L.orc_gdn_sequential.argtypes = [i64, i64, i64, i64, vp, vp, vp, vp, vp, ct.c_double, vp, vp, vp]
        L.orc_gdn_sequential.restype = ct.c_int
        L.orc_gdn_chunked.argtypes = [i64, i64, i64, i64, i64, vp, vp, vp, vp, vp, ct.c_double, vp, vp, vp, vp]
        L.orc_gdn_chunked.restype = ct.c_int
        L.orc_e4m3_decode.argtypes = [ct.c_uint8]
        L.orc_e4m3_decode.restype = ct.c_float
        L.orc_e4m3_encode.argtypes = [ct.c_float]
        L.orc_e4m3_encode.restype = ct.c_uint8
        L.orc_bf16_round.argtypes = [ct.c_float]
        L.orc_bf16_round.restype = ct.c_uint16
        L.orc_fp8_quantize.argtypes = [vp, vp, u64, ct.c_float]
        L.orc_fp8_dequantize.argtypes = [vp, vp, u64, ct.c_float]
        self.lib = L

    # ---- gated linear attention (§2 hybrid recurrent state; §5 chunking) ----
    @staticmethod
    def _check_inputs(q, k, v, g):
        for a in (q, k, v, g):
            if a.dtype != np.float32 or not a.flags.c_contiguous:
                raise TypeError("oracle inputs must be C-contiguous float32")
        T, H, dk = q.shape
        if k.shape != (T, H, dk) or v.shape[:2] != (T, H) or g.shape != (T, H):
            raise ValueError("shape mismatch")
        return T, H, dk, v.shape[2]

    def sequential(self, q, k, v, g, S0=None, scale=1.0):
        """Token-by-token recurrence S_t = exp(g_t) S_{t-1} + k_t^T v_t,
        o_t = scale * q_t S_t.  Returns (o [T,H,dv] f64, S_final [H,dk,dv] f64)."""
        T, H, dk, dv = self._check_inputs(q, k, v, g)
        S0 = None if S0 is None else np.ascontiguousarray(S0, dtype=np.float64)
        if S0 is not None and S0.shape != (H, dk, dv):
            raise ValueError("S0 shape")
        o = np.empty((T, H, dv), np.float64)
        S = np.empty((H, dk, dv), np.float64)
        rc = self.lib.orc_linattn_sequential(T, H, dk, dv, _ptr(q), _ptr(k), _ptr(v), _ptr(g),
                                             float(scale), _ptr(S0), _ptr(o), _ptr(S))
        if rc != 0:
            raise ValueError("orc_linattn_sequential failed")
        return o, S

    def chunked(self, q, k, v, g, chunk, S0=None, scale=1.0, want_chunk_states=True):
        """Chunked form with chunk size ``chunk`` (§5).  Returns
        (o [T,H,dv], chunk_states [ceil(T/C),H,dk,dv] or None, S_final [H,dk,dv]),
        all fp64; chunk_states[j] is the state entering chunk j."""
        T, H, dk, dv = self._check_inputs(q, k, v, g)
        S0 = None if S0 is None else np.ascontiguousarray(S0, dtype=np.float64)
        if S0 is not None and S0.shape != (H, dk, dv):
            raise ValueError("S0 shape")
        n_chunks = (T + chunk - 1) // chunk
        o = np.empty((T, H, dv), np.float64)
        cs = np.empty((n_chunks, H, dk, dv), np.float64) if want_chunk_states else None
        S = np.empty((H, dk, dv), np.float64)
        rc = self.lib.orc_linattn_chunked(T, H, dk, dv, int(chunk), _ptr(q), _ptr(k), _ptr(v), _ptr(g),
                                          float(scale), _ptr(S0), _ptr(o), _ptr(cs), _ptr(S))
        if rc != 0:
            raise ValueError("orc_linattn_chunked failed")
        return o, cs, S

    # ---- gated delta rule (the model's Gated DeltaNet state; reading in gdn_oracle.c) ----
    def _gdn_check(self, q, k, v, g, beta):
        T, H, dk, dv = self._check_inputs(q, k, v, g)
        if not (isinstance(beta, np.ndarray) and beta.dtype == np.float32 and beta.flags.c_contiguous
                and beta.shape == (T, H)):
            raise ValueError("beta must be a C-contiguous float32 [T, H] array")
        return T, H, dk, dv

    def gdn_sequential(self, q, k, v, g, beta, S0=None, scale=1.0):
        """S_t = exp(g_t)(I - beta_t k_t^T k_t) S_{t-1} + beta_t k_t^T v_t, o_t = scale q_t S_t,
        token by token.  Returns (o [T,H,dv] f64, S_final [H,dk,dv] f64)."""
        T, H, dk, dv = self._gdn_check(q, k, v, g, beta)
        S0 = None if S0 is None else np.ascontiguousarray(S0, dtype=np.float64)
        o = np.empty((T, H, dv), np.float64)
        S = np.empty((H, dk, dv), np.float64)
        if self.lib.orc_gdn_sequential(T, H, dk, dv, _ptr(q), _ptr(k), _ptr(v), _ptr(g), _ptr(beta), float(scale),
                                       _ptr(S0), _ptr(o), _ptr(S)) != 0:
            raise ValueError("orc_gdn_sequential failed")
        return o, S

    def gdn_chunked(self, q, k, v, g, beta, chunk, S0=None, scale=1.0):
        """The chunked (WY) form with chunk size ``chunk``.  Returns
        (o, chunk_states [ceil(T/C),H,dk,dv] (state entering each chunk), S_final), fp64."""
        T, H, dk, dv = self._gdn_check(q, k, v, g, beta)
        S0 = None if S0 is None else np.ascontiguousarray(S0, dtype=np.float64)
        n_chunks = (T + chunk - 1) // chunk
        o = np.empty((T, H, dv), np.float64)
        cs = np.empty((n_chunks, H, dk, dv), np.float64)
        S = np.empty((H, dk, dv), np.float64)
        if self.lib.orc_gdn_chunked(T, H, dk, dv, int(chunk), _ptr(q), _ptr(k), _ptr(v), _ptr(g), _ptr(beta),
                                    float(scale), _ptr(S0), _ptr(o), _ptr(cs), _ptr(S)) != 0:
            raise ValueError("orc_gdn_chunked failed")
        return o, cs, S

    # ---- capsule verbs as memcpy (§3 Algorithm 1, "Four verbs") ----
    def align(self, P, C):
        """P' = floor(P / C) * C (§3 Algorithm 1)."""
        return int(self.lib.orc_align(int(P), int(C)))

    @staticmethod
    def _layout(row_bytes, rows_total, kinds):
        rb = np.ascontiguousarray(row_bytes, dtype=np.uint64)
        rt = np.ascontiguousarray(rows_total, dtype=np.uint64)
        kd = np.ascontiguousarray(kinds, dtype=np.uint32)
        if not (len(rb) == len(rt) == len(kd)):
            raise ValueError("layout length mismatch")
        return rb, rt, kd

    def capsule_bytes(self, row_bytes, rows_total, kinds, P_aligned):
        rb, rt, kd = self._layout(row_bytes, rows_total, kinds)
        return int(self.lib.orc_capsule_bytes(len(rb), _ptr(rb), _ptr(rt), _ptr(kd), int(P_aligned)))

    @staticmethod
    def _ptr_array(arrays):
        return (ct.c_void_p * len(arrays))(*[a.ctypes.data for a in arrays])

    def snapshot(self, bufs, row_bytes, rows_total, kinds, P_aligned):
        """Return the capsule bytes (uint8 array) of host buffers ``bufs``."""
        rb, rt, kd = self._layout(row_bytes, rows_total, kinds)
        for b in bufs:
            assert b.flags.c_contiguous
        n = int(self.lib.orc_capsule_bytes(len(rb), _ptr(rb), _ptr(rt), _ptr(kd), int(P_aligned)))
        arena = np.empty(n, np.uint8)
        self.lib.orc_capsule_snapshot(len(rb), self._ptr_array(bufs), _ptr(rb), _ptr(rt), _ptr(kd),
                                      int(P_aligned), _ptr(arena))
        return arena

    def restore(self, arena, bufs, row_bytes, rows_total, kinds, P_aligned):
        """Copy capsule bytes back into host buffers ``bufs`` (in place)."""
        rb, rt, kd = self._layout(row_bytes, rows_total, kinds)
        arena = np.ascontiguousarray(arena, dtype=np.uint8)
        self.lib.orc_capsule_restore(len(rb), self._ptr_array(bufs), _ptr(rb), _ptr(rt), _ptr(kd),
                                     int(P_aligned), _ptr(arena))

    def append(self, bufs, srcs, row_bytes, rows_total, kinds, position, n):
        """Append n rows at ``position`` into host buffers ``bufs`` (in place):
        positional buffers get rows [position, position + n) from their source,
        fixed buffers slide as windows; ``srcs[i]`` None leaves buffer i alone.
        Returns the oracle's status (0, or -1 if a positional buffer is full)."""
        rb, rt, kd = self._layout(row_bytes, rows_total, kinds)
        keep = [None if x is None else np.ascontiguousarray(x) for x in srcs]
        src_arr = (ct.c_void_p * len(srcs))(*[None if x is None else x.ctypes.data for x in keep])
        width = max([int(rb[i] * (rt[i] + n)) for i in range(len(rb))] + [1])
        scratch = np.empty(width, np.uint8)
        return int(self.lib.orc_set_append(len(rb), self._ptr_array(bufs), src_arr, _ptr(rb), _ptr(rt), _ptr(kd),
                                           int(position), int(n), _ptr(scratch)))

    def fork(self, arena, sets, row_bytes, rows_total, kinds, P_aligned):
        """Restore the same capsule into each buffer list of ``sets``."""
        rb, rt, kd = self._layout(row_bytes, rows_total, kinds)
        flat = [b for s in sets for b in s]
        self.lib.orc_capsule_fork(len(rb), len(sets), self._ptr_array(flat), _ptr(rb), _ptr(rt), _ptr(kd),
                                  int(P_aligned), _ptr(np.ascontiguousarray(arena, dtype=np.uint8)))

    def gather(self, gallery, ids, sets, row_bytes, rows_total, kinds, P_aligned):
        """Environment e receives gallery[ids[e]] (a list of uint8 arenas)."""
        rb, rt, kd = self._layout(row_bytes, rows_total, kinds)
        flat = [b for s in sets for b in s]
        ids = np.ascontiguousarray(ids, dtype=np.int32)
        gal = self._ptr_array([np.ascontiguousarray(a, dtype=np.uint8) for a in gallery])
        rc = self.lib.orc_capsule_gather(len(rb), len(sets), self._ptr_array(flat), _ptr(rb), _ptr(rt),
                                         _ptr(kd), int(P_aligned), len(gallery), gal, _ptr(ids))
        if rc != 0:
            raise ValueError("gallery id out of range")

    def digest_tokens(self, ids):
        """64-bit FNV-1a over the little-endian bytes of int32 token ids."""
        ids = np.ascontiguousarray(ids, dtype=np.int32)
        return int(self.lib.orc_digest_tokens(_ptr(ids), len(ids)))

    def digest_bytes(self, data: bytes):
        buf = (ct.c_ubyte * max(1, len(data))).from_buffer_copy(data or b"\0")
        return int(self.lib.orc_digest_bytes(ct.cast(buf, ct.c_void_p), len(data)))


    # ---- FP8 KV region (§3 "Definition": FP8-KV halves the KV region; the
    # BF16 working stage is rebuilt lazily, §3 cost model).  OCP E4M3.
    def e4m3_decode(self, code: int) -> float:
        return float(self.lib.orc_e4m3_decode(int(code) & 0xFF))

    def e4m3_encode(self, x: float) -> int:
        return int(self.lib.orc_e4m3_encode(float(np.float32(x))))

    def bf16_round(self, y: float) -> int:
        return int(self.lib.orc_bf16_round(float(np.float32(y))))

    def fp8_quantize(self, src_bf16_bits, scale):
        """uint16 bf16 bit patterns -> uint8 E4M3 codes of x / scale."""
        src = np.ascontiguousarray(src_bf16_bits, dtype=np.uint16)
        out = np.empty(src.shape, dtype=np.uint8)
        self.lib.orc_fp8_quantize(_ptr(src), _ptr(out), src.size, float(np.float32(scale)))
        return out

    def fp8_dequantize(self, codes, scale):
        """uint8 E4M3 codes -> uint16 bf16 bit patterns of decode(code) * scale."""
        src = np.ascontiguousarray(codes, dtype=np.uint8)
        out = np.empty(src.shape, dtype=np.uint16)
        self.lib.orc_fp8_dequantize(_ptr(src), _ptr(out), src.size, float(np.float32(scale)))
        return out


_default = None


def get(rebuild: bool = False) -> Oracle:
    """The default oracle build (compiled on first use if absent)."""
    global _default
    if _default is None or rebuild:
        if rebuild or not os.path.exists(_build.LIB_PATH):
            _build.build()
        _default = Oracle(_build.LIB_PATH)
    return _default
