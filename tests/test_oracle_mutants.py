"""The pins catch plausible mistakes in the oracle.

Each case copies the oracle's C sources to a temporary directory, plants one
mistake by a textual substitution (a dropped term, a wrong sign, a wrong index,
a transposed operand, a wrong constant), builds that copy with gcc and runs the
pin suite against it: at least one pin must fail.  Mistakes are chosen so that
the mutated code still stays inside its buffers.
"""
import os
import shutil

import pytest

import oracle
from oracle import build as obuild
from oracle_pins import CAPSULE_PINS, FP8_PINS, GDN_PINS, SCAN_PINS

ORACLE_DIR = os.path.dirname(os.path.abspath(oracle.__file__))

MUTANTS = [
    # (id, file, old text, new text, pin family)
    ("seq_dropped_decay", "linattn_oracle.c",
     "S[i * dv + j] = decay * S[i * dv + j] + ki", "S[i * dv + j] = S[i * dv + j] + ki", "scan"),
    ("seq_k_replaced_by_q", "linattn_oracle.c",
     "const double ki = (double)AT3(k, t, h, i, H, dk);",
     "const double ki = (double)AT3(q, t, h, i, H, dk);", "scan"),
    ("seq_head_index_dropped_in_S0", "linattn_oracle.c",
     "S[i] = S0 ? S0[h * dk * dv + i] : 0.0;\n        for (int64_t t = 0;",
     "S[i] = S0 ? S0[i] : 0.0;\n        for (int64_t t = 0;", "scan"),
    ("chunk_mask_drops_diagonal", "linattn_oracle.c",
     "for (int64_t m = 0; m <= i; ++m)", "for (int64_t m = 0; m < i; ++m)", "scan"),
    ("chunk_decay_sign", "linattn_oracle.c",
     "exp(G[i] - G[m]) * qk", "exp(G[m] - G[i]) * qk", "scan"),
    ("chunk_inter_decay_dropped", "linattn_oracle.c",
     "inter[j] = exp(G[i]) * acc;", "inter[j] = acc;", "scan"),
    ("chunk_state_decay_wrong_index", "linattn_oracle.c",
     "const double chunk_decay = exp(G[L - 1]);", "const double chunk_decay = exp(G[0]);", "scan"),
    ("chunk_exclusive_cumsum", "linattn_oracle.c",
     "run += (double)g[(t0 + i) * H + h];\n                G[i] = run;",
     "G[i] = run;\n                run += (double)g[(t0 + i) * H + h];", "scan"),
    ("chunk_fold_weight_dropped", "linattn_oracle.c",
     "const double w = exp(G[L - 1] - G[m]);", "const double w = 1.0;", "scan"),
    ("chunk_scale_twice", "linattn_oracle.c",
     "AT3(o, ti, h, j, H, dv) *= scale;", "AT3(o, ti, h, j, H, dv) *= scale * scale;", "scan"),
    ("chunk_fold_uses_q", "linattn_oracle.c",
     "const double kd = w * (double)AT3(k, tm, h, d, H, dk);",
     "const double kd = w * (double)AT3(q, tm, h, d, H, dk);", "scan"),
    ("align_rounds_up", "capsule_oracle.c",
     "return C ? (P / C) * C : 0;", "return C ? ((P + C - 1) / C) * C : 0;", "capsule"),
    ("positional_copies_all_rows", "capsule_oracle.c",
     "return kind == ORC_KIND_POSITIONAL ? P_aligned * row_bytes : row_bytes * rows_total;",
     "return row_bytes * rows_total;", "capsule"),
    ("fnv_wrong_prime", "capsule_oracle.c",
     "h *= 1099511628211ULL;", "h *= 1099511628213ULL;", "capsule"),
    ("gather_ignores_ids", "capsule_oracle.c",
     "gallery[ids[e]]);", "gallery[e % n_gallery]);", "capsule"),
    ("append_window_keeps_oldest", "capsule_oracle.c",
     "memcpy(dst, scratch + n * rb, (size_t)(W * rb));", "memcpy(dst, scratch, (size_t)(W * rb));", "capsule"),
    ("append_positional_off_by_one", "capsule_oracle.c",
     "memcpy(dst + position * rb, srcs[i], (size_t)(n * rb));",
     "memcpy(dst + (position + 1) * rb, srcs[i], (size_t)((n - 1) * rb));", "capsule"),
    ("gdn_seq_correction_sign", "gdn_oracle.c",
     "a * (S[i * dv + j] - b * ki * kS[j])", "a * (S[i * dv + j] + b * ki * kS[j])", "gdn"),
    ("gdn_seq_correction_without_beta", "gdn_oracle.c",
     "a * (S[i * dv + j] - b * ki * kS[j])", "a * (S[i * dv + j] - ki * kS[j])", "gdn"),
    ("gdn_seq_decay_after_correction", "gdn_oracle.c",
     "a * (S[i * dv + j] - b * ki * kS[j])", "a * S[i * dv + j] - b * ki * kS[j]", "gdn"),
    ("gdn_chunk_solve_sign", "gdn_oracle.c",
     "for (int64_t j = 0; j < t; ++j) acc -= A[t * C + j] * W[j * dk + d];",
     "for (int64_t j = 0; j < t; ++j) acc += A[t * C + j] * W[j * dk + d];", "gdn"),
    ("gdn_chunk_w_without_gamma", "gdn_oracle.c",
     "double acc = bt * gt * (double)AT3(k, t0 + t, h, d, H, dk);",
     "double acc = bt * (double)AT3(k, t0 + t, h, d, H, dk);", "gdn"),
    ("gdn_chunk_mask_drops_diagonal", "gdn_oracle.c",
     "for (int64_t j = 0; j <= t; ++j) {", "for (int64_t j = 0; j < t; ++j) {", "gdn"),
    ("gdn_chunk_fold_weight_dropped", "gdn_oracle.c",
     "acc += exp(G[L - 1] - G[j]) * (double)AT3(k, t0 + j, h, d, H, dk) * U[j * dv + e];",
     "acc += (double)AT3(k, t0 + j, h, d, H, dk) * U[j * dv + e];", "gdn"),
    ("e4m3_bias_off_by_one", "fp8_oracle.c",
     "return ldexp(1.0 + (double)m / 8.0, (int)e - 7);", "return ldexp(1.0 + (double)m / 8.0, (int)e - 8);", "fp8"),
    ("e4m3_subnormal_scale", "fp8_oracle.c",
     "return ldexp((double)m / 8.0, -6);", "return ldexp((double)m / 8.0, -7);", "fp8"),
    ("e4m3_ties_to_odd", "fp8_oracle.c",
     "(d == best_d && (c & 1u) == 0u)", "(d == best_d && (c & 1u) == 1u)", "fp8"),
    ("e4m3_overflow_to_nan", "fp8_oracle.c",
     "if (a >= 448.0) return (uint8_t)(sign | 0x7Eu);", "if (a >= 448.0) return (uint8_t)(sign | 0x7Fu);", "fp8"),
    ("fp8_quantize_multiplies_by_scale", "fp8_oracle.c",
     "const float x = bf16_value(src_bf16[i]) * inv;", "const float x = bf16_value(src_bf16[i]) * scale;", "fp8"),
    ("fp8_dequantize_drops_scale", "fp8_oracle.c",
     "const float y = orc_e4m3_decode(c) * scale;", "const float y = orc_e4m3_decode(c);", "fp8"),
    ("bf16_ties_away", "fp8_oracle.c",
     "return (uint16_t)(((lo >> 16) & 1u) ? (hi >> 16) : (lo >> 16));", "return (uint16_t)(hi >> 16);", "fp8"),
]


@pytest.mark.parametrize("mid,fname,old,new,family", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_mutant_is_caught(tmp_path, mid, fname, old, new, family):
    src = tmp_path / "src"
    src.mkdir()
    for s in obuild.SOURCES:
        shutil.copy(os.path.join(ORACLE_DIR, s), src / s)
    text = (src / fname).read_text()
    assert old in text, "mutation anchor no longer present in %s: %r" % (fname, old)
    (src / fname).write_text(text.replace(old, new))
    lib = obuild.build(out_path=str(tmp_path / ("liborc_%s.so" % mid)), src_dir=str(src))
    mutant = oracle.Oracle(lib)
    pins = {"scan": SCAN_PINS, "capsule": CAPSULE_PINS, "fp8": FP8_PINS, "gdn": GDN_PINS}[family]
    caught = []
    for pin in pins:
        try:
            pin(mutant)
        except (AssertionError, ValueError):
            caught.append(pin.__name__)
    assert caught, "mutant %s passed every pin" % mid
