"""Planted mistakes in the C oracle: each altered copy of oracle/caffe_ref.c
must fail at least one of the oracle's pins (tests/test_oracle_conv.py,
tests/test_oracle_glue.py), so that a plausible slip anywhere in the oracle
-- a flipped kernel, a dropped bias, a wrong mask, index, sign or divisor --
cannot pass them.  CPU only: each mutant is compiled with gcc into a
temporary directory and the pins run against it through
oracle.ref.library().  The unaltered source, built the same way, must pass
every pin (the control)."""
import inspect
import os
import shutil
import subprocess

import pytest

import oracle.ref as ref
import test_oracle_conv
import test_oracle_glue

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "caffe_ref.c")

# (name, original text, planted text, occurrences replaced)
MUTANTS = [
    ("kernel flip (convolution instead of cross-correlation)",
     "z += w[((k * Cg + c) * kh + u) * kw + v] *",
     "z += w[((k * Cg + c) * kh + (kh - 1 - u)) * kw + (kw - 1 - v)] *", 1),
    ("dropped bias", "double z = b ? b[k] : 0.0;", "double z = 0.0;", 1),
    (">= ReLU mask in the backward pass", "if (relu && !(top[idx] > 0.0))",
     "if (relu && !(top[idx] >= 0.0))", 1),
    ("wrong group slice in the forward gather",
     "z += w[((k * Cg + c) * kh + u) * kw + v] *\n"
     "                                     x[((n * C + t * Cg + c) * H + ih) * W + iw];",
     "z += w[((k * Cg + c) * kh + u) * kw + v] *\n"
     "                                     x[((n * C + c) * H + ih) * W + iw];", 1),
    ("transposed taps", "z += w[((k * Cg + c) * kh + u) * kw + v] *",
     "z += w[((k * Cg + c) * kh + v) * kw + u] *", 1),
    ("pad sign", "const long ih = i * sh - ph + u;", "const long ih = i * sh + ph + u;", 3),
    ("weight-gradient taps transposed", "dwk[(c * kh + u) * kw + v] +=",
     "dwk[(c * kh + v) * kw + u] +=", 1),
    ("data-gradient scatter with the flipped filter",
     "dxs[(c * H + ih) * W + iw] +=\n"
     "                                            w[((k * Cg + c) * kh + u) * kw + v] * d;",
     "dxs[(c * H + ih) * W + iw] +=\n"
     "                                            w[((k * Cg + c) * kh + (kh - 1 - u)) * kw +"
     " (kw - 1 - v)] * d;", 1),
    ("bias gradient without the ReLU mask",
     "s += masked_diff(top, top_diff, ((n * K + k) * Ho + i) * Wo + j, relu);",
     "s += top_diff[((n * K + k) * Ho + i) * Wo + j];", 1),
    ("max-pool tie to the last maximum", "plane[h * W + ww] > bv", "plane[h * W + ww] >= bv", 1),
    ("max-pool backward overwrites instead of summing",
     "dplane[a] += top_diff[(nc * Ho + i) * Wo + j];",
     "dplane[a] = top_diff[(nc * Ho + i) * Wo + j];", 1),
    ("LRN divisor dropped", "return kk + alpha / size * sq;", "return kk + alpha * sq;", 1),
    ("LRN window shifted", "long a = c - (size - 1) / 2, b = a + size;",
     "long a = c - (size - 1) / 2 + 1, b = a + size;", 1),
    ("LRN exponent sign", "y[(n * C + c) * HW + e] = col[c * HW] * pow(s, -beta);",
     "y[(n * C + c) * HW + e] = col[c * HW] * pow(s, beta);", 1),
    ("LRN backward cross-term sign",
     "gcol[c * HW] * pow(s_c, -beta) - 2.0 * alpha * beta / size",
     "gcol[c * HW] * pow(s_c, -beta) + 2.0 * alpha * beta / size", 1),
]


def _pins():
    """Every pin of the two oracle test modules, parametrizations expanded:
    (label, function, keyword arguments)."""
    out = []
    for mod in (test_oracle_conv, test_oracle_glue):
        for name, f in vars(mod).items():
            if not name.startswith("test_") or not callable(f):
                continue
            combos = [{}]
            for m in getattr(f, "pytestmark", []):
                if m.name != "parametrize":
                    continue
                names = m.args[0]
                names = [a.strip() for a in names.split(",")] if isinstance(names, str) else names
                new = []
                for c in combos:
                    for v in m.args[1]:
                        v = getattr(v, "values", v)
                        vals = (v,) if len(names) == 1 else tuple(v)
                        d = dict(c)
                        d.update(zip(names, vals))
                        new.append(d)
                combos = new
            for c in combos:
                out.append((f"{mod.__name__}.{name}{c or ''}", f, c))
    return out


def _run_pin(f, kwargs, golden_dir):
    if "golden_dir" in inspect.signature(f).parameters:
        kwargs = dict(kwargs, golden_dir=golden_dir)
    f(**kwargs)


def _build(src_text, d):
    c = os.path.join(d, "caffe_ref.c")
    so = os.path.join(d, "libcaffe_ref.so")
    with open(c, "w") as fh:
        fh.write(src_text)
    subprocess.run(["gcc", "-O1", "-std=c11", "-fopenmp", "-fPIC", "-shared", c, "-o", so, "-lm"],
                   check=True, capture_output=True)
    return so


needs_gcc = pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not found")


@needs_gcc
def test_unaltered_copy_passes_every_pin(tmp_path, golden_dir):
    so = _build(open(SRC).read(), str(tmp_path))
    with ref.library(so):
        for label, f, kw in _pins():
            _run_pin(f, kw, golden_dir)


@needs_gcc
@pytest.mark.parametrize("mutant", MUTANTS, ids=[m[0] for m in MUTANTS])
def test_planted_mistake_fails_a_pin(mutant, tmp_path, golden_dir):
    name, old, new, count = mutant
    src = open(SRC).read()
    assert src.count(old) == count, f"{name}: the original text occurs {src.count(old)} times"
    so = _build(src.replace(old, new), str(tmp_path))
    caught = None
    with ref.library(so):
        for label, f, kw in _pins():
            try:
                _run_pin(f, kw, golden_dir)
            except (AssertionError, ValueError) as e:
                caught = (label, type(e).__name__)
                break
    assert caught is not None, f"planted mistake '{name}' passed every pin"
    print(f"{name}: caught by {caught[0]}")
