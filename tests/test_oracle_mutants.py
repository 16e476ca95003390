"""The pins catch plausible mistakes in the oracle: each mutant below is the
oracle's source with one mistake planted (on the CPU, in a temporary copy),
built and loaded in a fresh pytest process that runs the pin tests; every
mutant must make at least one pin fail, and the unmodified source must pass."""
import os
import subprocess
import sys

import pytest

from oracle import build as ob

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PINS = [os.path.join(ROOT, "tests", f) for f in ("test_oracle_pins.py", "test_oracle_fv_pins.py")]

# (name, text in zo_oracle.c, replacement) -- each text occurs exactly once
MUTANTS = [
    ("l1-left-to-right", "    return tree_abs(a, n, next_pow2(n));",
     "    float t = 0.0f; for (int64_t j = 0; j < n; ++j) t += fabsf(a[j]); return t;"),
    ("scale-divisor", "    float s = l1 / (float)n;", "    float s = l1 / (float)(n + 1);"),
    ("sign-of-zero", "bit[j] = (a[j] >= 0.0f) ? 1 : 0;", "bit[j] = (a[j] > 0.0f) ? 1 : 0;"),
    ("worker-error-sign", "            delta[base + j] = bit[j] ? (a[j] - s) : (a[j] + s);",
     "            delta[base + j] = bit[j] ? (a[j] + s) : (a[j] - s);"),
    ("pack-msb-first", "if (bit[j]) words[j / 64] |= (uint64_t)1 << (j % 64);",
     "if (bit[j]) words[j / 64] |= (uint64_t)1 << (63 - j % 64);"),
    ("average-rounded-twice", "    *out = (float)(sum / (double)W);",
     "    *out = (float)sum / (float)W;"),
    ("server-error-sign", "            srv_delta[e] = bit[j] ? (b[j] - s) : (b[j] + s);",
     "            srv_delta[e] = bit[j] ? (b[j] + s) : (b[j] - s);"),
    ("server-error-dropped", "            b[j] = a + srv_delta[e];", "            b[j] = a;"),
    ("old-momentum", "        float m_used = p->literal_momentum ? m_old : m_new;",
     "        float m_used = m_old;"),
    ("buffer-not-accumulated", "        st->u[j] = st->u[j] + step;", "        st->u[j] = step;"),
    ("sync-from-model", "        st->x[j] = st->anchor[j] - ubar[j] / den;",
     "        st->x[j] = st->x[j] - ubar[j] / den;"),
    ("momentum-divisor", "        st->m[j] = ubar[j] / gsum;", "        st->m[j] = ubar[j];"),
    ("gamma-sum-kept", "    }\n    st->gamma_sum = 0.0f;\n}", "    }\n}"),
    ("variance-abs", "        st->v[j] = p->beta2 * st->v[j] + p->c2 * (gbar[j] * gbar[j]);",
     "        st->v[j] = p->beta2 * st->v[j] + p->c2 * fabsf(gbar[j]);"),
    ("fv-new-momentum", "        float step = gamma * m_old;\n        float den = sqrtf(v_old + p->eps);\n        x[j]",
     "        float step = gamma * m[j];\n        float den = sqrtf(v_old + p->eps);\n        x[j]"),
    ("fv-variance-always", "        if (update_v) v[j] =", "        v[j] ="),
    ("dense-average-worker-index", "            double term = (double)z[(int64_t)w * n + j];",
     "            double term = (double)z[(int64_t)j * W + w];"),
    ("dense-average-first-worker-only", "            double term = (double)z[(int64_t)w * n + j];",
     "            double term = (double)z[j];"),
]


def _run_pins(lib):
    env = dict(os.environ, ZO_ORACLE_LIB=lib)
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        "-m", "not gpu"] + PINS, cwd=ROOT, env=env, capture_output=True,
                       text=True, timeout=300)
    return r.returncode, r.stdout[-2000:]


def _build(tmp_path, text):
    src = tmp_path / "zo_oracle.c"
    src.write_text(text)
    return ob.build(src=str(src), out=str(tmp_path / "liboracle.so"))


def test_unmodified_source_passes(tmp_path):
    text = open(os.path.join(ob.HERE, "zo_oracle.c")).read()
    rc, out = _run_pins(_build(tmp_path, text))
    assert rc == 0, out


@pytest.mark.parametrize("name,old,new", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_mutant_is_caught(tmp_path, name, old, new):
    text = open(os.path.join(ob.HERE, "zo_oracle.c")).read()
    assert text.count(old) == 1, f"{name}: the text to mutate must occur once"
    rc, out = _run_pins(_build(tmp_path, text.replace(old, new)))
    assert rc == 1, f"mutant {name} survived the pins:\n{out}"
