"""Mutation check of the oracle's pins: each case plants one plausible
mistake in a copy of the C oracle (a dropped term, a wrong sign, index,
constant, rounding or comparison), builds that copy with the oracle's own
flags, and runs the pin suites against it in a child process.  Every
mutant must make at least one pin fail; a mutant that passes them all marks
a part of the oracle that nothing outside the oracle checks.

The planted mistakes follow the places where the method can be misread:
the equations of motion and the explicit Euler update (Sec. "Cart-pole
environment"), the termination rule, the counter-based generator and the
way its words become actions and start states, the MLP policy, and the
binary64/binary16 variants of the step."""
import concurrent.futures as cf
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

from oracle import build as obuild  # noqa: E402

PIN_FILES = ["tests/test_oracle_pins.py", "tests/test_oracle_precision.py"]

# name: (text in cartpole_oracle.c, replacement); each text occurs once.
MUTANTS = {
    # binary32 dynamics
    "gravity_sign": ("(g * sn - c * temp) / (l * (four3 - mp * c2 / m));\n    const float xacc",
                     "(-g * sn - c * temp) / (l * (four3 - mp * c2 / m));\n    const float xacc"),
    "thd_not_squared": ("const float thd2 = thd * thd;", "const float thd2 = thd;"),
    "missing_pml_c": ("const float xacc = temp - pml * thacc * c / m;",
                      "const float xacc = temp - pml * thacc / m;"),
    "semi_implicit_euler": (
        "out[0] = x + tau * xd;\n    out[1] = xd + tau * xacc;\n"
        "    out[2] = th + tau * thd;\n    out[3] = thd + tau * thacc;\n}\n\n/* The same",
        "out[1] = xd + tau * xacc;\n    out[0] = x + tau * out[1];\n"
        "    out[3] = thd + tau * thacc;\n    out[2] = th + tau * out[3];\n}\n\n/* The same"),
    # binary32 termination
    "obs_before_reset": ("                orc_reset_state(reset_seed, env, k, next);\n            }\n            memcpy(s, next, sizeof s);\n\n            if (obs)\n                for (int j = 0; j < 4; ++j) obs[(step * 4 + j) * m + i] = s[j];",
                         "                orc_reset_state(reset_seed, env, k, s);\n            }\n            if (!d) memcpy(s, next, sizeof s);\n\n            if (obs)\n                for (int j = 0; j < 4; ++j) obs[(step * 4 + j) * m + i] = next[j];"),
    "no_reward_on_termination": ("int d = orc_terminated_f32(next);\n            float r = 1.0f;",
                                 "int d = orc_terminated_f32(next);\n            float r = d ? 0.0f : 1.0f;"),
    "length_kept_after_termination": ("                len = 0u;\n                k += 1u;\n                orc_reset_state(",
                                      "                k += 1u;\n                orc_reset_state("),
    "return_excludes_terminal_step": (
        "                returns += len;\n                n_done += 1u;\n                len = 0u;\n"
        "                k += 1u;\n                orc_reset_state(",
        "                returns += len - 1u;\n                n_done += 1u;\n                len = 0u;\n"
        "                k += 1u;\n                orc_reset_state("),
    "reset_keyed_by_old_episode": ("                k += 1u;\n                orc_reset_state(reset_seed, env, k, next);",
                                   "                orc_reset_state(reset_seed, env, k, next);\n                k += 1u;"),
    "terminated_on_old_state": ("            int d = orc_terminated_f32(next);", "            int d = orc_terminated_f32(s);"),
    "threshold_decimal": ("(float)(12.0 * 2.0 * 3.14159265358979323846 / 360.0)", "0.20944f"),
    "ge_not_gt": ("const float x_limit = 2.4f;", "const float x_limit = 2.4f * 0.9999999f;"),
    # generator, actions, start states
    "threefry_rotation": ("{13, 15, 26, 6, 17, 29, 16, 24}", "{13, 15, 26, 6, 17, 29, 16, 25}"),
    "threefry_parity": ("0x1BD11BDAu", "0x1BD11BDBu"),
    "threefry_injection": ("x1 += ks[(s + 1) % 3] + s;", "x1 += ks[(s + 1) % 3];"),
    "action_words_swapped": ("(j < 32u) ? w[0] : w[1]", "(j < 32u) ? w[1] : w[0]"),
    "action_bits_reversed": ("(word >> (j % 32u)) & 1u", "(word >> (31u - j % 32u)) & 1u"),
    "action_counter_swapped": ("orc_threefry2x32(key[0], key[1], env / 64u, t, w);",
                               "orc_threefry2x32(key[0], key[1], t, env / 64u, w);"),
    "stream_tags_swapped": ("#define ORC_TAG_ACTION 1u\n#define ORC_TAG_RESET 2u",
                            "#define ORC_TAG_ACTION 2u\n#define ORC_TAG_RESET 1u"),
    "seed_words_swapped": ("orc_threefry2x32((uint32_t)(seed >> 32), (uint32_t)seed, tag, 0u, key);",
                           "orc_threefry2x32((uint32_t)seed, (uint32_t)(seed >> 32), tag, 0u, key);"),
    "reset_halves_order": (
        "const uint32_t half[4] = {u[0] & 0xFFFFu, u[0] >> 16, u[1] & 0xFFFFu, u[1] >> 16};\n"
        "    const float scale",
        "const uint32_t half[4] = {u[0] >> 16, u[0] & 0xFFFFu, u[1] & 0xFFFFu, u[1] >> 16};\n"
        "    const float scale"),
    "reset_not_centred": ("int32_t centred = (int32_t)half[j] - (int32_t)(1 << 15);",
                          "int32_t centred = (int32_t)half[j] - (int32_t)(1 << 14);"),
    "reset_scale": ("ldexpf(0.1f, -16)", "ldexpf(0.1f, -15)"),
    "reset_counter_step": ("orc_reset_state(reset_seed, env, k, next);",
                           "orc_reset_state(reset_seed, env, t, next);"),
    # MLP policy
    "mlp_transpose": ("w[i * n_out + j]", "w[j * n_in + i]"),
    "mlp_no_bf16_input": ("in[i] = orc_f32_from_bf16(orc_bf16_from_f32(obs[i]));",
                          "in[i] = obs[i];"),
    "mlp_no_bf16_first_hidden": (
        "h1[j] = orc_f32_from_bf16(orc_bf16_from_f32((float)tanh((double)z1[j])));",
        "h1[j] = (float)tanh((double)z1[j]);"),
    "mlp_tie_picks_one": ("return z3[1] > z3[0] ? 1 : 0;", "return z3[1] >= z3[0] ? 1 : 0;"),
    "mlp_binary32_sums": ("        double acc = 0.0;", "        float acc = 0.0f;"),
    "bf16_truncates": ("u += 0x7FFFu + lsb;", "u += 0u * lsb;"),
    "bf16_ties_away": ("u += 0x7FFFu + lsb;", "u += 0x8000u + 0u * lsb;"),
    "mlp_no_bf16_hidden": (
        "h2[j] = orc_f32_from_bf16(orc_bf16_from_f32((float)tanh((double)z2[j])));",
        "h2[j] = (float)tanh((double)z2[j]);"),
    # binary64
    "f64_missing_c": ("const double xacc = temp - pml * thacc * c / m;",
                      "const double xacc = temp - pml * thacc / m;"),
    "f64_gravity_sign": ("const double thacc = (g * sn - c * temp) / (l * (four3 - mp * c2 / m));",
                         "const double thacc = (-g * sn - c * temp) / (l * (four3 - mp * c2 / m));"),
    "f64_semi_implicit_euler": (
        "const double xacc = temp - pml * thacc * c / m;\n\n    out[0] = x + tau * xd;\n"
        "    out[1] = xd + tau * xacc;",
        "const double xacc = temp - pml * thacc * c / m;\n\n    out[1] = xd + tau * xacc;\n"
        "    out[0] = x + tau * out[1];"),
    "f16_gravity_sign": ("const double thacc = h(h(h(g * sn) - h(c * temp))",
                         "const double thacc = h(h(h(-g * sn) - h(c * temp))"),
    "f16_semi_implicit_euler": ("    out[2] = h(th + h(tau * thd));\n    out[3] = h(thd + h(tau * thacc));",
                                "    out[3] = h(thd + h(tau * thacc));\n    out[2] = h(th + h(tau * out[3]));"),
    "f16_unrounded_cosine": ("const double c = h(cos(th));", "const double c = cos(th);"),
    "f64_reset_scale_single": ("ldexp(0.1, -16)", "ldexp((double)0.1f, -16)"),
    "f64_threshold_single": (
        "const double x_limit = 2.4, th_limit = 12.0 * 2.0 * 3.14159265358979323846 / 360.0;",
        "const double x_limit = 2.4, th_limit = (float)(12.0 * 2.0 * 3.14159265358979323846 / 360.0);"),
    # binary16
    "f16_ties_away": ("nearbyint(a / q)", "round(a / q)"),
    "f16_no_subnormal_floor": ("if (qexp < -24) qexp = -24;", "if (qexp < -30) qexp = -30;"),
    "f16_overflow_at_max": ("if (a >= 65520.0)", "if (a > 65504.0)"),
    "f16_unrounded_square": ("h(thd * thd)", "(thd * thd)"),
    "f16_unrounded_mass": ("const double m = h(mp + mc);", "const double m = mp + mc;"),
    "f16_unrounded_threshold": ("th_limit = h(12.0 * 2.0 * 3.14159265358979323846 / 360.0)",
                                "th_limit = (12.0 * 2.0 * 3.14159265358979323846 / 360.0)"),
}


def _source():
    with open(obuild.SRC) as f:
        return f.read()


def test_each_mutation_site_occurs_once():
    src = _source()
    for name, (old, _) in MUTANTS.items():
        assert src.count(old) == 1, name


def _run_mutant(name, src, tmpdir):
    old, new = MUTANTS[name]
    c_path = os.path.join(tmpdir, f"{name}.c")
    so_path = os.path.join(tmpdir, f"lib{name}.so")
    with open(c_path, "w") as f:
        f.write(src.replace(old, new))
    subprocess.run(["gcc", *obuild.CFLAGS, c_path, "-o", so_path, "-lm"], check=True,
                   capture_output=True)
    env = dict(os.environ, ORACLE_LIB=so_path, PYTHONDONTWRITEBYTECODE="1")
    r = subprocess.run([sys.executable, "-m", "pytest", *PIN_FILES, "-q", "-x",
                        "-p", "no:cacheprovider", "-m", "not gpu"],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    last = (r.stdout.strip().splitlines() or [""])[-1]
    return r.returncode, last


def test_unmutated_copy_passes_the_pins(tmp_path):
    """The harness itself: the same build route with no mutation passes."""
    src = _source()
    so_path = str(tmp_path / "liborig.so")
    c_path = str(tmp_path / "orig.c")
    with open(c_path, "w") as f:
        f.write(src)
    subprocess.run(["gcc", *obuild.CFLAGS, c_path, "-o", so_path, "-lm"], check=True)
    env = dict(os.environ, ORACLE_LIB=so_path, PYTHONDONTWRITEBYTECODE="1")
    r = subprocess.run([sys.executable, "-m", "pytest", *PIN_FILES, "-q", "-x",
                        "-p", "no:cacheprovider", "-m", "not gpu"],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    assert r.returncode == 0, r.stdout[-2000:]


def test_every_mutant_fails_a_pin(tmp_path):
    src = _source()
    workers = max(1, min(6, (os.cpu_count() or 2) - 2))
    with cf.ThreadPoolExecutor(workers) as ex:
        futs = {name: ex.submit(_run_mutant, name, src, str(tmp_path)) for name in MUTANTS}
        results = {name: f.result() for name, f in futs.items()}
    survivors = {name: last for name, (rc, last) in results.items() if rc == 0}
    assert not survivors, f"mutants no pin caught: {survivors}"
    # a failing run must be a test failure (rc 1), not a crash of the harness
    crashed = {name: (rc, last) for name, (rc, last) in results.items() if rc not in (0, 1)}
    assert not crashed, crashed
