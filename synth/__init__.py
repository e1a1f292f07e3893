"""Seeded synthetic inputs and the workload table.

This module is shared, as data, by the CPU oracle runs and the device runs.
It draws random numbers and encodes them (bf16 rounding, per-token L2
normalisation, the log-sigmoid gate transform); it holds none of the scan's or
the capsule's arithmetic.

Generator: numpy ``Generator(PCG64(SeedSequence([...])))``; every tensor has
its own stream, keyed by (workload seed, layer, tensor name).  Distributions
follow the workload descriptions: q, k ~ N(0,1) then L2-normalised per token
and head over dk (in fp64, no epsilon) and rounded to the input dtype;
v ~ N(0,1); log-gate g = log(sigmoid(x)), x ~ N(3, 0.5), computed in fp64 as
-log1p(exp(-x)) and rounded to fp32; delta-rule write strength beta =
sigmoid(x), x ~ N(0, 1), in fp64 rounded to fp32; KV rows, conv tails and denoiser state
~ N(0,1).
"""
from .configs import CONFIGS, Workload, get_config  # noqa: F401
from .gen import (  # noqa: F401
    bf16_bits,
    bf16_from_bits,
    bf16_round,
    fill_normal_bytes,
    gdn_inputs,
    linattn_inputs,
    normal_tensor,
    rng,
    token_ids,
)
