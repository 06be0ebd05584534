"""Mutation check of the oracle's pins (CPU only).

Each case plants one plausible mistake in a copy of the oracle's C source (a transposed operand,
a dropped term, a wrong exponent bias, a missing sign, a wrong rounding tie, a dropped softmax
scale or normaliser, a wrong slice ...), builds it into a temporary library, and runs the pin
suite against it in a subprocess.  The pins must reject every mutant.
"""
import os
import shutil
import subprocess
import sys

import pytest

import oracle

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "nmm_oracle.c")

MUTANTS = {
    "gemv_transposed_w": ("double p = dec(dt, x[m * ldx + k]) * dec(dt, W[k * ldw + n]);",
                          "double p = dec(dt, x[m * ldx + k]) * dec(dt, W[(n % K) * ldw + (k % N)]);"),
    "gemv_drops_last_term": ("for (int64_t k = 0; k < K; ++k) {\n            double p",
                             "for (int64_t k = 0; k + 1 < K; ++k) {\n            double p"),
    "gemv_abs_without_fabs": ("sa += fabs(p);", "sa += p;"),
    "bf16_bias_off_by_one": ("ldexp((double)(128 + f), e - 134)", "ldexp((double)(128 + f), e - 133)"),
    "bf16_sign_dropped": ("v = ldexp((double)(128 + f), e - 134);  /* (1 + f/2^7) * 2^(e-127) */\n    }\n    return sign ? -v : v;",
                          "v = ldexp((double)(128 + f), e - 134);  /* (1 + f/2^7) * 2^(e-127) */\n    }\n    return v;"),
    "f16_subnormal_scale": ("ldexp((double)f, -24)", "ldexp((double)f, -25)"),
    "rne_ties_away": ("return (fmod(fl, 2.0) == 0.0) ? fl : fl + 1.0;", "return fl + 1.0;"),
    "batched_ignores_x_stride": ("nmmo_gemv(M, K, N, dt, x + b * stride_x,", "nmmo_gemv(M, K, N, dt, x,"),
    "attention_drops_scale": ("s[j] = scale * acc;", "s[j] = acc;"),
    "attention_unnormalised": ("out[h * ldo + n] = o / l;", "out[h * ldo + n] = o;"),
    "attention_v_shifted": ("double v = nmmo_dec_bf16(kv[j * ldkv + n]);",
                            "double v = nmmo_dec_bf16(kv[j * ldkv + (n + 1) % dv]);"),
    "round_away_ignored": ("    if (mode == NMMO_ROUND_AWAY) return fl + 1.0;\n", ""),
    "round_away_breaks_down": ("    if (mode == NMMO_ROUND_AWAY) return fl + 1.0;", "    if (mode == NMMO_ROUND_AWAY) return fl;"),
    "rmsnorm_sum_not_mean": ("double inv = 1.0 / sqrt(ss / (double)n + eps);", "double inv = 1.0 / sqrt(ss + eps);"),
    "rmsnorm_drops_eps": ("double inv = 1.0 / sqrt(ss / (double)n + eps);", "double inv = 1.0 / sqrt(ss / (double)n);"),
    "rmsnorm_ignores_gamma": ("out[i] = c[i] * inv * nmmo_dec_bf16(gamma[i]);", "out[i] = c[i] * inv;"),
    "rope_turns_backwards": ("out[2 * i] = k[2 * i] * cs - k[2 * i + 1] * sn;\n        out[2 * i + 1] = k[2 * i] * sn + k[2 * i + 1] * cs;",
                             "out[2 * i] = k[2 * i] * cs + k[2 * i + 1] * sn;\n        out[2 * i + 1] = -k[2 * i] * sn + k[2 * i + 1] * cs;"),
    "rope_half_exponent": ("pow(theta, -2.0 * (double)i / (double)d)", "pow(theta, -(double)i / (double)d)"),
    "rope_rotates_halves": ("out[2 * i] = k[2 * i] * cs - k[2 * i + 1] * sn;\n        out[2 * i + 1] = k[2 * i] * sn + k[2 * i + 1] * cs;",
                            "out[i] = k[i] * cs - k[i + d / 2] * sn;\n        out[i + d / 2] = k[i] * sn + k[i + d / 2] * cs;"),
    "kv_entry_rope_on_latent": ("nmmo_rope(rope, mm + kv_lora, t, theta, r + kv_lora);", "nmmo_rope(rope, mm, t, theta, r + kv_lora);"),
    "kv_entry_fixed_mode": ("nmmo_round_bf16_array(r, row_bf16, kv_lora + rope, mode);", "nmmo_round_bf16_array(r, row_bf16, kv_lora + rope, 0);"),
    "kv_update_wrong_pitch": ("h, hidden, w, ldw, mm, mm_abs, n, nthreads);", "h, hidden, w, n, mm, mm_abs, n, nthreads);"),
    "chain_takes_rope_slice": ("b[h * nope + d] = nmmo_round_bf16_rne((float)buf[h * (nope + rope) + d]);",
                               "b[h * nope + d] = nmmo_round_bf16_rne((float)buf[h * (nope + rope) + rope + d]);"),
}


@pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not available")
@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_reject_mutant(name, tmp_path):
    old, new = MUTANTS[name]
    src = open(SRC).read()
    assert src.count(old) == 1, f"mutation site for {name} not found exactly once"
    msrc = tmp_path / "mutant.c"
    msrc.write_text(src.replace(old, new))
    so = oracle.build(force=True, src=str(msrc), out=str(tmp_path / "libmutant.so"))
    env = dict(os.environ, NMM_ORACLE_LIB=so, OMP_NUM_THREADS="2")
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        os.path.join(ROOT, "tests", "test_oracle_pins.py"),
                        os.path.join(ROOT, "tests", "test_alg2_schedule.py")],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=300)
    assert r.returncode != 0, f"mutant {name} passed every pin:\n{r.stdout[-2000:]}"
