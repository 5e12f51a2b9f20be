"""Planted-mistake check of the oracle's pins.

Each entry plants one plausible mistake in a copy of the oracle (the C
half, or the Python decoding loop), builds that copy, and runs the pin
suite against it in a subprocess: at least one pin must fail.  A mistake
that no pin catches would mean the pins do not fix that part of what the
oracle computes.  The mistakes are planted in copies on the CPU only; the
oracle itself is never changed.
"""
import concurrent.futures as cf
import os
import shutil
import subprocess
import sys
import tempfile

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
ORACLE_C = os.path.join(ROOT, "oracle", "oracle.c")
ORACLE_PY = os.path.join(ROOT, "oracle", "__init__.py")
PINS = ["tests/test_oracle_pins.py", "tests/test_follow_route.py"]

# (name, file, text in the oracle, planted replacement)
MUTATIONS = [
    ("rope_sign", "c", "x[i] = (float)((double)a * c - (double)b * s);",
     "x[i] = (float)((double)a * c + (double)b * s);"),
    ("norm_denominator", "c", "double r = 1.0 / sqrt(ss / n + eps);",
     "double r = 1.0 / sqrt(ss / (n - 1) + eps);"),
    ("causal_length", "c", "orc_attend(q, K, V, pos[r] + 1, dh, out);",
     "orc_attend(q, K, V, pos[r] + (pos[r] > 0 ? 0 : 1), dh, out);"),
    ("attention_scale", "c", "double scale = 1.0 / sqrt((double)dh);",
     "double scale = 1.0 / (double)dh;"),
    ("topk_tie_to_higher_id", "c",
     "if (!taken[e] && (best < 0 || logits[e] > logits[best])) best = e;",
     "if (!taken[e] && (best < 0 || logits[e] >= logits[best])) best = e;"),
    ("swiglu_operands_swapped", "c", "(float)(silu(g[i]) * (double)u[i])",
     "(float)(silu(u[i]) * (double)g[i])"),
    ("moe_norm_gain_of_attention", "c",
     "orc_rmsnorm(h + (size_t)r * H, w->ffn_norm + (size_t)layer * H, H, d->rms_eps,",
     "orc_rmsnorm(h + (size_t)r * H, w->attn_norm + (size_t)layer * H, H, d->rms_eps,"),
    ("gate_weight_dropped", "c", "const float c = (float)((double)p * tmp[(size_t)t * H + i]);",
     "const float c = (float)((double)tmp[(size_t)t * H + i]);"),
    ("argmax_tie_to_higher_id", "c", "if (lg[v] > lg[best]) best = v;",
     "if (lg[v] >= lg[best]) best = v;"),
    ("kv_not_rounded", "c", "kd[t] = st_in(d, k[hh * dh + t]);", "kd[t] = k[hh * dh + t];"),
    ("input_row_shifted", "c",
     "for (int r = 0; r < nr; ++r) input_row(d, w, tok[r], emb, r, h + (size_t)r * H);",
     "for (int r = 0; r < nr; ++r) input_row(d, w, tok[r > 0 ? r - 1 : 0], emb, r > 0 ? r - 1 : 0, h + (size_t)r * H);"),
    ("draft_output_norm", "c",
     "orc_rmsnorm(z + (size_t)r * H, w->final_norm, H, d->rms_eps, u + (size_t)r * H);",
     "orc_rmsnorm(z + (size_t)r * H, w->d_ffn_norm, H, d->rms_eps, u + (size_t)r * H);"),
    ("draft_concat_order", "c",
     "orc_rmsnorm(e, w->d_enorm, H, d->rms_eps, c);\n    orc_rmsnorm(a + (size_t)r * H, w->d_hnorm, H, d->rms_eps, c + H);",
     "orc_rmsnorm(e, w->d_enorm, H, d->rms_eps, c + H);\n    orc_rmsnorm(a + (size_t)r * H, w->d_hnorm, H, d->rms_eps, c);"),
    ("residual_dropped", "c", "for (size_t i = 0; i < (size_t)nr * H; ++i) h[i] = (float)((double)h[i] + proj[i]);",
     "for (size_t i = 0; i < (size_t)nr * H; ++i) h[i] = proj[i];"),
    ("follow_tolerance_sign", "c", "if (min_in >= max_out - tol) {", "if (min_in >= max_out + tol) {"),
    ("follow_accepts_duplicates", "c", "if (given[u] == given[t]) return 1;",
     "if (given[u] == given[t] && 0) return 1;"),
    ("follow_accepts_past_end", "c", "if (given[t] < 0 || given[t] >= E) return 1;",
     "if (given[t] < 0 || given[t] > E) return 1;"),
    ("commit_wrong_bonus", "py", "commit = [int(t) for t in draft[:m]] + [int(verify[m])]",
     "commit = [int(t) for t in draft[:m]] + [int(verify[max(m - 1, 0)])]"),
    ("catchup_rows_short", "py", "    st.n_rows = m + 1\n",
     "    st.n_rows = max(m, 1)\n"),
    ("chain_position", "py", "        p = st.row_pos + n - 1 + (d - 1)\n",
     "        p = st.row_pos + n - 1 + d\n"),
]


def _plant(tmp, kind, old, new):
    """A broken copy of the oracle in tmp; returns the subprocess env."""
    env = dict(os.environ, OMP_NUM_THREADS="1", PYTHONDONTWRITEBYTECODE="1")
    src = open(ORACLE_C if kind == "c" else ORACLE_PY).read()
    assert src.count(old) == 1, f"planted text not found exactly once: {old!r}"
    if kind == "c":
        path = os.path.join(tmp, "oracle.c")
        open(path, "w").write(src.replace(old, new))
        lib = os.path.join(tmp, "_oracle_mut.so")
        subprocess.check_call(["gcc", "-O2", "-fPIC", "-shared", "-fopenmp", "-std=c11", path,
                               "-o", lib, "-lm"])
        env["MTP_ORACLE_LIB"] = lib
    else:
        pkg = os.path.join(tmp, "oracle")
        os.makedirs(pkg)
        open(os.path.join(pkg, "__init__.py"), "w").write(src.replace(old, new))
        env["MTP_ORACLE_LIB"] = os.path.join(ROOT, "oracle", "_oracle.so")
    return env


# the broken copy is imported before pytest puts the repository on the path
_DRIVER = """
import sys
tmp, root = sys.argv[1], sys.argv[2]
sys.path.insert(0, root)
sys.path.insert(0, tmp)
import oracle
assert oracle.__file__.startswith(tmp) or not __import__("os").path.isdir(tmp + "/oracle")
import pytest
sys.exit(pytest.main(sys.argv[3:]))
"""


def _pins_fail(kind, old, new):
    tmp = tempfile.mkdtemp(prefix="orc_mut_")
    try:
        env = _plant(tmp, kind, old, new)
        r = subprocess.run([sys.executable, "-c", _DRIVER, tmp, ROOT, *PINS, "-x", "-q",
                            "-p", "no:cacheprovider", "-m", "not slow"],
                           cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
        return r.returncode, r.stdout[-400:]
    finally:
        shutil.rmtree(tmp, ignore_errors=True)


@pytest.fixture(scope="module")
def outcomes():
    import oracle
    oracle.build(force=False)
    with cf.ThreadPoolExecutor(max_workers=min(8, os.cpu_count() or 1)) as ex:
        futs = {m[0]: ex.submit(_pins_fail, m[1], m[2], m[3]) for m in MUTATIONS}
        return {k: f.result() for k, f in futs.items()}


@pytest.mark.parametrize("name", [m[0] for m in MUTATIONS])
def test_planted_mistake_fails_a_pin(outcomes, name):
    rc, tail = outcomes[name]
    assert rc == 1, f"no pin caught the planted mistake {name} (rc {rc}):\n{tail}"


def test_unmutated_copy_passes():
    """The harness itself: a copy with no change passes every pin."""
    rc, tail = _pins_fail("c", "#include <math.h>", "#include <math.h>")
    assert rc == 0, tail
