"""The oracle's pins reject plausible mistakes in it.

Each case plants one mistake in a copy of oracle/oracle.c (a textual replacement
that must match exactly once), builds it with the oracle's own compiler line, and
runs the pin suite tests/test_oracle.py against it (ORACLE_LIB): the suite must
fail.  A control build of the unchanged source must pass.  Nothing here touches the
oracle itself."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "oracle.c")

# name -> (text in oracle.c, replacement)
MUTANTS = {
    "keep_rule_strict": ("        keep[r] = z <= w[r];", "        keep[r] = z < w[r];"),
    "count_strict": ("        n += z <= w[r];", "        n += z < w[r];"),
    "missing_2pi": ("double lambda = two_pi / th; /* +inf when th == 0 */",
                    "double lambda = 1.0 / th; /* +inf when th == 0 */"),
    "exponent_sign": ("        double th = theta ? theta[r] : pow(base, -2.0 * (double)r / (double)d);\n"
                      "        if (!(th >= 0.0))\n            return -1;\n        double lambda",
                      "        double th = theta ? theta[r] : pow(base, 2.0 * (double)r / (double)d);\n"
                      "        if (!(th >= 0.0))\n            return -1;\n        double lambda"),
    "dropped_scale": ("    return x * scale;", "    return x;"),
    "interleaved_pairs": ("qd[r + h] * load_elem(k, krow_off + r + h, kdt)",
                          "qd[r + 1] * load_elem(k, krow_off + r + 1, kdt)"),
    "gqa_map": ("            const int64_t g = hq / group;", "            const int64_t g = hq % h_kv;"),
    "causal_off_by_one": ("const int64_t last = p < n_k - 1 ? p : n_k - 1; /* causal: keys j <= p */",
                          "const int64_t last = p - 1 < n_k - 1 ? p - 1 : n_k - 1; /* causal */"),
    "distance_sign": ("(double)(p - j), w, atom, scale,\n                                  &kept);",
                      "(double)(j - p), w, atom, scale,\n                                  &kept);"),
    "count_ceil": ("            const double lo = (double)p - floor(w[r]);",
                   "            const double lo = (double)p - ceil(w[r]);"),
    "lse_log2": ("            lse_out[t] = m + log(l);", "            lse_out[t] = m + log2(l);"),
    "softmax_no_max": ("                const double e = exp(s[j] - m);",
                       "                const double e = exp(s[j]);"),
    "rounded_slice_high_freq": ("        keep[r] = r >= h - nr;", "        keep[r] = r < nr;"),
    "distance_count_length": ("        retained += (uint64_t)(hi - lo + 1) * (uint64_t)kept;",
                              "        retained += (uint64_t)(hi - lo) * (uint64_t)kept;"),
    "family_floor": ("        if (w < beta)\n            w = beta;", "        if (w > beta)\n            w = beta;"),
}


def _build(tmp_path, text, name):
    c = tmp_path / f"{name}.c"
    so = tmp_path / f"lib{name}.so"
    c.write_text(text)
    subprocess.run(["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c11", "-o", str(so),
                    str(c), "-lm"], check=True, capture_output=True)
    return str(so)


def _pins(so):
    env = dict(os.environ, ORACLE_LIB=so, OMP_NUM_THREADS="4")
    return subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                           os.path.join(ROOT, "tests", "test_oracle.py")],
                          cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)


def test_control_build_passes_the_pins(tmp_path):
    r = _pins(_build(tmp_path, open(SRC).read(), "control"))
    assert r.returncode == 0, r.stdout[-2000:]


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_pins_reject_planted_mistake(tmp_path, name):
    old, new = MUTANTS[name]
    src = open(SRC).read()
    assert src.count(old) == 1, f"{name}: the text to mutate must occur exactly once"
    r = _pins(_build(tmp_path, src.replace(old, new), name))
    assert r.returncode == 1 and " failed" in r.stdout, \
        f"{name}: the pins did not catch it\n{r.stdout[-1500:]}"
