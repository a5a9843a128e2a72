"""The oracle's pins must be strong enough to catch plausible mistakes.

Each case plants one mistake in a copy of the oracle's C source (a dropped
term, a wrong sign, a swapped index, a wrong rounding, an off-by-one), builds
it, and runs the oracle pin suite against that build: the suite must fail.
Everything runs on the CPU; the real oracle is never modified.  (Replacing the
strict "norm > clip" by ">=" is not listed: at norm == clip both give a
coefficient of exactly 1, so that mutant is equivalent.)
"""
import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "zero_oracle.c")
PIN_TESTS = ["tests/test_oracle_accounting.py", "tests/test_oracle_layout.py", "tests/test_oracle_binary16.py",
             "tests/test_oracle_stats.py", "tests/test_oracle_adam.py", "tests/test_oracle_invariants.py",
             "tests/test_oracle_lamb.py", "tests/test_oracle_scaler.py"]

MUTANTS = {
    "update_sign": ("float th = theta[i] - h->lr * u;", "float th = theta[i] + h->lr * u;"),
    "bias_correction_swapped": ("float mhat = mi / h->bc1;", "float mhat = mi / h->bc2;"),
    "eps_inside_sqrt": ("float denom = sqrtf(vhat) + h->eps;", "float denom = sqrtf(vhat + h->eps);"),
    "variance_not_squared": ("h->omb2 * (g * g);", "h->omb2 * g;"),
    "variance_decay_beta1": ("float vi = h->b2 * *v", "float vi = h->b1 * *v"),
    "bias_t_off_by_one": ("h->bc1 = (float)(1.0 - pow(beta1, (double)t));",
                          "h->bc1 = (float)(1.0 - pow(beta1, (double)(t + 1)));"),
    "no_bias_correction_v": ("h->bc2 = (float)(1.0 - pow(beta2, (double)t));", "h->bc2 = 1.0f;"),
    "decay_sign": ("u = u + h->wd * theta;", "u = u - h->wd * theta;"),
    "clip_inverted": ("clip / out->norm : 1.0;", "out->norm / clip : 1.0;"),
    "unscale_multiplies": ("out->mult = (float)(out->coef / loss_scale);",
                           "out->mult = (float)(out->coef * loss_scale);"),
    "norm_keeps_scale": ("out->norm = sqrt(out->sumsq) / loss_scale;", "out->norm = sqrt(out->sumsq);"),
    "nan_not_overflow": ("if ((h & 0x7C00u) == 0x7C00u) {", "if ((h & 0x7FFFu) == 0x7C00u) {"),
    "units_shift": ("return (1024u + f) << (e - 1);", "return (1024u + f) << e;"),
    "subnormal_decode": ("mag = ldexp((double)f, -24);", "mag = ldexp((double)f, -25);"),
    "round_ties_away": ("(frac == 0.5 && fmod(k, 2.0) != 0.0)", "(frac == 0.5)"),
    "round_truncates": ("if (frac > 0.5 || (frac == 0.5 && fmod(k, 2.0) != 0.0))", "if (0)"),
    "layout_floor": ("        S += 1;\n", "        S += 0;\n"),
    "layout_valid_unclamped": ("    if (valid > S)\n        valid = S;\n", ""),
    "pos_g_forgets_grads": ("case 2: return 2.0 * psi + (2.0 + k) * psi / nd;",
                            "case 2: return 2.0 * psi + k * psi / nd;"),
    "writes_on_skip": ("    if (sc.skip)\n        return 1;\n", ""),
    "scaler_no_halving": ("double s = *scale / 2.0;", "double s = *scale;"),
    "t_counts_skips": ("        *good = 0;\n        return;\n", "        *good = 0;\n        *applied += 1;\n        return;\n"),
    "scaler_growth_late": ("*good >= window", "*good > window"),
    "scaler_skip_keeps_good": ("        *good = 0;\n        return;\n", "        return;\n"),
    # exact fp32 sum of squares
    "acc_drops_carry": ("        if (i - q >= 1 && carry == 0)\n", "        if (i - q >= 1)\n"),
    "acc_carry_not_added": ("zo_u128 s = (zo_u128)a->limb[i] + carry + (i - q < 2 ? parts[i - q] : 0);",
                            "zo_u128 s = (zo_u128)a->limb[i] + (i - q < 2 ? parts[i - q] : 0);"),
    "acc_ignores_sticky": ("(rem == 0x400u && (sticky || (mant & 1u)))", "(rem == 0x400u && (mant & 1u))"),
    "acc_ties_away": ("(rem == 0x400u && (sticky || (mant & 1u)))", "(rem == 0x400u)"),
    "acc_subnormal_exponent": ("int E = e ? (int)e - 150 : -149;", "int E = e ? (int)e - 150 : -150;"),
    "acc_implicit_bit": ("uint64_t M = e ? (f | 0x800000u) : f;", "uint64_t M = f;"),
    # LAMB
    "lamb_trust_inverted": ("trust = wn / sqrt(su);", "trust = sqrt(su) / wn;"),
    "lamb_weight_norm_squared": ("double wn = sqrt(st);", "double wn = st;"),
    "lamb_zero_norm_freezes": ("        double trust = 1.0;\n", "        double trust = 0.0;\n"),
    "lamb_phi_upper_uses_lower": ("            if (wn > phi_hi)\n                wn = phi_hi;\n",
                                  "            if (wn > phi_hi)\n                wn = phi_lo;\n"),
    "lamb_phi_lower_ignored": ("            if (wn < phi_lo)\n                wn = phi_lo;\n", ""),
    "lamb_layer_tail_skipped": ("        for (int64_t j = 0; j < len; ++j) {\n            const int64_t i = a + j;\n            float g",
                                "        for (int64_t j = 0; j < len - 1; ++j) {\n            const int64_t i = a + j;\n            float g"),
    "lamb_writes_on_skip": ("    if (sc.skip != 0)\n        return 1;\n", ""),
    "lamb_applies_adam_step": ("float th = theta[i] - step * u[j];", "float th = theta[i] - h->lr * u[j];"),
    "lamb_norm_over_whole_vector": ("const double st = zo_sumsq_f32(theta + a, len);",
                                    "const double st = zo_sumsq_f32(theta, n);"),
}


def _build_mutant(tmp, name, old, new):
    src = open(SRC).read()
    assert src.count(old) == 1, name
    path = os.path.join(tmp, name + ".c")
    with open(path, "w") as f:
        f.write(src.replace(old, new))
    lib = os.path.join(tmp, name + ".so")
    subprocess.run(["gcc", "-std=gnu11", "-O2", "-ffp-contract=off", "-fno-fast-math", "-fPIC", "-shared",
                    "-w", path, "-o", lib, "-lm"], check=True)
    return lib


def _suite_fails(lib):
    env = dict(os.environ, ZERO_ORACLE_LIB=lib)
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider", "-k", "not exhaustive",
                        *PIN_TESTS],
                       cwd=ROOT, env=env, stdout=subprocess.PIPE, stderr=subprocess.STDOUT, timeout=600)
    return r.returncode != 0, r.stdout.decode(errors="replace")[-400:]


@pytest.mark.skipif(shutil.which("gcc") is None, reason="needs gcc")
def test_every_planted_mistake_is_caught(tmp_path):
    libs = {name: _build_mutant(str(tmp_path), name, old, new) for name, (old, new) in MUTANTS.items()}
    with ThreadPoolExecutor(max_workers=4) as ex:
        results = dict(zip(libs, ex.map(_suite_fails, libs.values())))
    survivors = {k: tail for k, (failed, tail) in results.items() if not failed}
    assert not survivors, survivors
