"""Seeded generators (no method arithmetic; see the package docstring)."""
import zlib

import numpy as np

_NAME_IDS = {}


def _name_id(name: str) -> int:
    if name not in _NAME_IDS:
        _NAME_IDS[name] = zlib.crc32(name.encode())
    return _NAME_IDS[name]


def rng(seed: int, layer: int, name: str, block: int = 0) -> np.random.Generator:
    """Independent PCG64 stream for (seed, layer, tensor name, block)."""
    ss = np.random.SeedSequence([int(seed), int(layer) & 0xFFFFFFFF, _name_id(name), int(block)])
    return np.random.Generator(np.random.PCG64(ss))


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 values to bfloat16 (round to nearest, ties to even) and
    return the 16-bit patterns as uint16.  Inputs must be finite."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    lsb = (u >> 16) & 1
    r = (u + 0x7FFF + lsb) >> 16
    return r.astype(np.uint16)


def bf16_from_bits(b: np.ndarray) -> np.ndarray:
    """Widen bfloat16 bit patterns (uint16) to the exactly equal float32 values."""
    b = np.ascontiguousarray(b, dtype=np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32)


def bf16_round(x: np.ndarray) -> np.ndarray:
    """float32 -> nearest bfloat16 value, returned as float32."""
    return bf16_from_bits(bf16_bits(x))


def normal_tensor(seed, layer, name, shape, dtype="bf16", block=0):
    """N(0,1) tensor.  Returns (values_f32, device_payload) where the payload is
    the uint16 bf16 patterns (dtype 'bf16') or the float32 values ('f32')."""
    x = rng(seed, layer, name, block).standard_normal(size=shape, dtype=np.float32)
    if dtype == "bf16":
        bits = bf16_bits(x)
        return bf16_from_bits(bits).reshape(shape), bits.reshape(shape)
    if dtype == "f32":
        return x, x
    raise ValueError(dtype)


def fill_normal_bytes(seed, layer, name, nbytes, block=0) -> np.ndarray:
    """nbytes of N(0,1) float32 payload (for byte-level buffers), as uint8."""
    assert nbytes % 4 == 0
    x = rng(seed, layer, name, block).standard_normal(size=nbytes // 4, dtype=np.float32)
    return x.view(np.uint8)


def _l2_normalise_rows(x64: np.ndarray) -> np.ndarray:
    n = np.sqrt(np.sum(x64 * x64, axis=-1, keepdims=True))
    return x64 / n


def linattn_inputs(seed: int, layer: int, T: int, H: int, dk: int, dv: int, dtype: str = "bf16",
                   gate_mu: float = 3.0, gate_sigma: float = 0.5, t_offset_block: int = 0):
    """q, k, v, g for one linear-attention layer.

    Returns a dict with float32 value arrays 'q','k','v' ([T,H,d]) and 'g'
    ([T,H]) -- the exact values the device sees -- plus 'q_dev','k_dev',
    'v_dev' payloads (uint16 bf16 patterns for dtype 'bf16', float32 for 'f32').
    """
    out = {}
    for name, d in (("q", dk), ("k", dk), ("v", dv)):
        r = rng(seed, layer, name, t_offset_block)
        x = r.standard_normal(size=(T, H, d))  # float64
        if name in ("q", "k"):
            x = _l2_normalise_rows(x)
        x32 = x.astype(np.float32)
        if dtype == "bf16":
            bits = bf16_bits(x32)
            out[name] = bf16_from_bits(bits).reshape(T, H, d)
            out[name + "_dev"] = bits.reshape(T, H, d)
        elif dtype == "f32":
            out[name] = x32
            out[name + "_dev"] = x32
        else:
            raise ValueError(dtype)
    r = rng(seed, layer, "g", t_offset_block)
    x = r.normal(gate_mu, gate_sigma, size=(T, H))
    out["g"] = (-np.log1p(np.exp(-x))).astype(np.float32)
    return out


def gdn_inputs(seed: int, layer: int, T: int, H: int, dk: int, dv: int, dtype: str = "bf16",
               gate_mu: float = 3.0, gate_sigma: float = 0.5, t_offset_block: int = 0):
    """linattn_inputs plus the write strengths 'beta' ([T,H] float32) of a
    delta-rule layer: beta = sigmoid(x), x ~ N(0, 1), computed in fp64 and
    rounded to fp32."""
    out = linattn_inputs(seed, layer, T, H, dk, dv, dtype, gate_mu, gate_sigma, t_offset_block)
    x = rng(seed, layer, "beta", t_offset_block).standard_normal(size=(T, H))
    out["beta"] = (1.0 / (1.0 + np.exp(-x))).astype(np.float32)
    return out


def token_ids(seed: int, n: int, vocab: int = 151_936) -> np.ndarray:
    """Synthetic int32 token ids (metadata for the prefix digest only)."""
    return rng(seed, 0, "tokens").integers(0, vocab, size=n, dtype=np.int32)
