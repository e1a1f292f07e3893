"""The five synthetic workloads, by their shapes and sizes.

Shapes follow the workload descriptions; readings of unstated details:
K and V are separate position-major buffers [T_max, kv_heads, d]; conv tails
are bf16 [width, channels] per linear layer; "2 MB" is 2 MiB; T_max is the
largest position used plus one chunk.
"""
from dataclasses import dataclass, field
from typing import Tuple


@dataclass(frozen=True)
class Workload:
    name: str
    seed: int
    n_linear: int            # gated linear-attention layers
    n_full: int              # full-attention layers (positional KV)
    heads: int               # linear-attention heads
    dk: int
    dv: int
    kv_heads: int
    kv_dim: int
    prefix: int              # snapshot boundary / prefill length
    chunk: int
    in_dtype: str            # 'bf16' or 'f32' for q, k, v
    kv_dtype_bytes: int
    t_max: int               # rows of each positional KV buffer
    conv_width: int = 0
    conv_channels: int = 0
    continuation: int = 0    # decode steps after the boundary
    extra: Tuple = field(default_factory=tuple)

    @property
    def kv_row_bytes(self) -> int:
        return self.kv_heads * self.kv_dim * self.kv_dtype_bytes

    @property
    def state_bytes(self) -> int:
        return self.heads * self.dk * self.dv * 4

    @property
    def conv_bytes(self) -> int:
        return self.conv_width * self.conv_channels * 2


CONFIGS = {
    # 1 linear layer, 2 heads, 64/64, T=256, chunk 64, fp32 q/k/v; one full-attn
    # KV buffer [512, 4, 64] bf16; snapshot at 128, continue to 256.
    "tiny": Workload("tiny", 20261202 + 0, n_linear=1, n_full=1, heads=2, dk=64, dv=64,
                     kv_heads=4, kv_dim=64, prefix=128, chunk=64, in_dtype="f32",
                     kv_dtype_bytes=2, t_max=512, continuation=128),
    # 6 linear + 2 full-attn layers, 16 heads 128/128, 4 KV heads d=128,
    # prefix 2048, chunk 64, conv tail 4 x 2048, then 32 continuation steps.
    "hybrid8": Workload("hybrid8", 20261202 + 1, n_linear=6, n_full=2, heads=16, dk=128, dv=128,
                        kv_heads=4, kv_dim=128, prefix=2048, chunk=64, in_dtype="bf16",
                        kv_dtype_bytes=2, t_max=8448, conv_width=4, conv_channels=2048,
                        continuation=32),
    # 36 linear + 12 full-attn layers, 32 heads 128/128, 4 KV heads d=256,
    # prefix 16384, chunk 64; cold prefill vs restore, fork into 4 sessions.
    "hybrid48": Workload("hybrid48", 20261202 + 2, n_linear=36, n_full=12, heads=32, dk=128, dv=128,
                         kv_heads=4, kv_dim=256, prefix=16384, chunk=64, in_dtype="bf16",
                         kv_dtype_bytes=2, t_max=16448, conv_width=4, conv_channels=4096,
                         continuation=1, extra=(("fork", 4),)),
    # hybrid8 shapes with boundaries at L, L+2, L+63 for L = 1k..8k.
    "align_stress": Workload("align_stress", 20261202 + 3, n_linear=6, n_full=2, heads=16, dk=128,
                             dv=128, kv_heads=4, kv_dim=128, prefix=2048, chunk=64, in_dtype="bf16",
                             kv_dtype_bytes=2, t_max=8448, conv_width=4, conv_channels=2048,
                             continuation=32,
                             extra=(("boundaries", (2048, 2050, 2111)),
                                    ("prefixes", tuple(range(1024, 8193, 1024))),
                                    ("offsets", (0, 2, 63)))),
    # Robot episode reset: 32 environments, gallery of 8 capsules, each = 18
    # layers of KV [816, 1, 256] bf16 (K and V) + 2 MiB fp32 denoiser state.
    "robot_reset": Workload("robot_reset", 20261202 + 4, n_linear=0, n_full=18, heads=0, dk=0, dv=0,
                            kv_heads=1, kv_dim=256, prefix=816, chunk=1, in_dtype="bf16",
                            kv_dtype_bytes=2, t_max=816,
                            extra=(("envs", 32), ("gallery", 8), ("resets", 1000),
                                   ("denoiser_bytes", 2 * 1024 * 1024))),
}


def get_config(name: str) -> Workload:
    return CONFIGS[name]
