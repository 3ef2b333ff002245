"""The oracle's pins have teeth: each plausible mistake below is planted in a
temporary copy of oracle/mot_oracle.c (CPU only), built with the same flags,
and the pins that guard that part of the definition are run against the
mutated build in a child process (MOT_ORACLE_LIB).  Every mutation must make
at least one of them fail; the unmutated build must pass them."""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "mot_oracle.c")

PINS = "tests/test_oracle_pins.py"
HAND = "tests/test_oracle_handworked.py"
USAGE = "tests/test_oracle_usage.py"
WINDOW = "tests/test_oracle_window.py"

# (name, original text, planted text, pins that must catch it); the original
# text must occur in the source, and every occurrence is replaced
MUTATIONS = [
    ("layernorm unbiased variance", "    var /= w;\n", "    var /= (w - 1);\n",
     [HAND + "::test_backbone_layernorms"]),
    ("layernorm eps outside the root", "1.0 / sqrt(var + 1e-5)", "1.0 / (sqrt(var) + 1e-5)",
     [HAND + "::test_backbone_layernorms"]),
    ("backbone attention scale 1/width", "sc[u] = acc / sqrt((double)hw);", "sc[u] = acc / (double)hw;",
     [HAND + "::test_backbone_attention_scale_and_heads"]),
    ("backbone attention scale over d_h", "sc[u] = acc / sqrt((double)hw);", "sc[u] = acc / sqrt((double)d_h);",
     [HAND + "::test_backbone_attention_scale_and_heads"]),
    ("backbone heads not split", "const double* qt = Q + (size_t)t * d_h + hh * hw;",
     "const double* qt = Q + (size_t)t * d_h;", [HAND + "::test_backbone_attention_scale_and_heads"]),
    ("replay attention scale 1/D", "const double scale = 1.0 / sqrt((double)D);",
     "const double scale = 1.0 / (double)D;", [HAND + "::test_replay_attention_scale"]),
    ("dropped layer-1 bias", "if (w->b1) acc += (double)w->b1[em * Hd + k];", "", [PINS]),
    ("no renormalisation over the Top-K set", "double gt = sel[m] ? g[m] / gsum : 0.0;",
     "double gt = sel[m] ? g[m] : 0.0;", [PINS]),
    ("Top-K ties to the higher index", "(best < 0 || g[m] > g[best])", "(best < 0 || g[m] >= g[best])", [PINS]),
    ("softmax sign flipped", "g[m] = exp(logits[m] - mx);", "g[m] = exp(mx - logits[m]);", [PINS]),
    ("tanh-form GELU in the oracle", "return 0.5 * a * (1.0 + erf(a / sqrt(2.0)));",
     "return 0.5 * a * (1.0 + tanh(0.7978845608028654 * (a + 0.044715 * a * a * a)));", [PINS]),
    ("transposed W1", "const float* w1 = w->w1 + (em * Hd + k) * d_in;\n            double acc = 0.0;\n"
     "            for (int32_t c = 0; c < d_in; ++c) acc += (double)w1[c] * z[c];",
     "const float* w1 = w->w1 + em * Hd * d_in + k;\n            double acc = 0.0;\n"
     "            for (int32_t c = 0; c < d_in; ++c) acc += (double)w1[(size_t)c * Hd] * z[c];", [PINS]),
    ("usage CV^2 with the sample variance", "    var /= E;\n", "    var /= (E - 1);\n", [USAGE]),
    ("usage entropy in bits", "h -= p * log(p);", "h -= p * log2(p);", [USAGE]),
    ("usage counts ties to the higher index", "if (!sel[m] && (best < 0 || g[m] > g[best])) best = m;\n"
     "                        sel[best] = 1;\n                    }\n                    for (int32_t m = 0; m < E; ++m) counts",
     "if (!sel[m] && (best < 0 || g[m] >= g[best])) best = m;\n"
     "                        sel[best] = 1;\n                    }\n                    for (int32_t m = 0; m < E; ++m) counts",
     [USAGE]),
    ("window scan starts from the last slot", "r == 0 ? z + (size_t)t * Nd_h :",
     "r == 0 ? z + (size_t)t * Nd_h + (size_t)(N - 1) * d_h :", [WINDOW]),
    ("window recurrence restarts from z_r",
     "r == 0 ? z + (size_t)t * Nd_h : F + (size_t)t * Nd_h + (size_t)(r - 1) * d_h",
     "z + (size_t)t * Nd_h + (size_t)r * d_h", [WINDOW]),
    ("window output LayerNorm per slot", "bb_layernorm(F + (size_t)t * Nd_h, Nd_h, ln_out_g, ln_out_b, t1);",
     "for (int32_t r2 = 0; r2 < N; ++r2) bb_layernorm(F + (size_t)t * Nd_h + (size_t)r2 * d_h, d_h, "
     "ln_out_g + (size_t)r2 * d_h, ln_out_b + (size_t)r2 * d_h, t1 + (size_t)r2 * d_h);", [WINDOW]),
    ("window router on the first slot only",
     "for (int32_t c = 0; c < Nd_in; ++c) acc += (double)wr[(unit * E + m) * Nd_in + c] * xt[c];",
     "for (int32_t c = 0; c < d_in; ++c) acc += (double)wr[(unit * E + m) * Nd_in + c] * xt[c];", [WINDOW]),
]


def _build(text, path):
    with open(path + ".c", "w") as f:
        f.write(text)
    subprocess.run(["gcc", "-O2", "-std=c99", "-ffp-contract=off", "-fno-fast-math", "-fPIC", "-shared", "-o", path,
                    path + ".c", "-lm", "-lpthread"], check=True)


def _run_pins(lib, pins):
    env = dict(os.environ, MOT_ORACLE_LIB=lib)
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider", *pins], cwd=ROOT,
                       env=env, capture_output=True, text=True, timeout=600)
    return r.returncode, r.stdout[-2000:]


@pytest.fixture(scope="module")
def original():
    return open(SRC).read()


def test_unmutated_build_passes(original, tmp_path):
    lib = str(tmp_path / "liboracle_same.so")
    _build(original, lib)
    pins = sorted({p for m in MUTATIONS for p in m[3]})
    rc, out = _run_pins(lib, pins)
    assert rc == 0, out


@pytest.mark.parametrize("name,old,new,pins", MUTATIONS, ids=[m[0] for m in MUTATIONS])
def test_mutation_is_caught(name, old, new, pins, original, tmp_path):
    assert old in original, name
    lib = str(tmp_path / "liboracle_mut.so")
    _build(original.replace(old, new), lib)
    rc, out = _run_pins(lib, pins)
    assert rc == 1, (name, rc, out)   # 1: tests ran and at least one failed
