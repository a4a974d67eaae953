"""Planted mistakes: each test compiles a copy of the oracle with one
plausible error written into it (on the CPU, in a temporary directory) and
checks that the pins reject that copy.  This shows the pins can tell a right
oracle from a wrong one."""
import os
import subprocess

import pytest

import oracle.oracle as orc
import pins

SRC = os.path.join(os.path.dirname(orc.__file__), "conv_oracle.c")

# (name, text to find, replacement, which occurrence (0-based))
PLANTS = [
    ("fwd kernel flipped",
     "double wv = w[((k * t->cg + cc) * t->r + r) * t->s + s];\n                acc += xv * wv;",
     "double wv = w[((k * t->cg + cc) * t->r + (t->r - 1 - r)) * t->s + (t->s - 1 - s)];\n"
     "                acc += xv * wv;", 0),
    ("fwd pad sign", "int64_t i = p * t->sh - t->ph + r * t->dh;",
     "int64_t i = p * t->sh + t->ph + r * t->dh;", 0),
    ("fwd dropped last tap", "for (int64_t r = 0; r < t->r; ++r)\n            for (int64_t s = 0; s < t->s; ++s) {\n                int64_t i",
     "for (int64_t r = 0; r < t->r - 1; ++r)\n            for (int64_t s = 0; s < t->s; ++s) {\n                int64_t i", 0),
    ("fwd ignores group offset", "double xv = x_at(t, x, n, gk * t->cg + cc, i, j);\n                double wv",
     "double xv = x_at(t, x, n, cc, i, j);\n                double wv", 0),
    ("x rows and columns swapped", "return x[((n * t->c + c) * t->h + i) * t->w + j];",
     "return x[((n * t->c + c) * t->h + j % t->h) * t->w + i % t->w];", 0),
    ("dgrad ignores stride divisibility", "if (num_p < 0 || num_p % t->sh != 0) continue;",
     "if (num_p < 0) continue;", 0),
    ("dgrad upper bound off by one", "if (q >= t->q) continue;\n                double dyv",
     "if (q >= t->q - 1) continue;\n                double dyv", 0),
    ("dgrad weight channel index reversed",
     "double wv = w[((k * t->cg + cc) * t->r + r) * t->s + s];\n                acc += dyv * wv;",
     "double wv = w[((k * t->cg + (t->cg - 1 - cc)) * t->r + r) * t->s + s];\n"
     "                acc += dyv * wv;", 0),
    ("wgrad ignores dilation", "int64_t i = p * t->sh - t->ph + r * t->dh;\n                int64_t j = q * t->sw - t->pw + s * t->dw;\n                double xv = x_at(t, x, n, gk * t->cg + cc, i, j);\n                double dyv",
     "int64_t i = p * t->sh - t->ph + r;\n                int64_t j = q * t->sw - t->pw + s * t->dw;\n                double xv = x_at(t, x, n, gk * t->cg + cc, i, j);\n                double dyv", 0),
    ("wgrad drops loss scale", "dwt[e] = old + inv_loss_scale * raw;", "dwt[e] = old + raw;", 0),
    ("wgrad ignores accumulate", "double old = beta ? dwt[e] : 0.0;", "double old = 0.0;", 0),
    ("output size rounds up", "t->p = num_h / sh + 1;", "t->p = (num_h + sh - 1) / sh + 1;", 0),
    ("nonfinite check misses NaN", "if (!isfinite(v[e])) return 1;", "if (isinf(v[e])) return 1;", 0),
]


def _planted_lib(tmp_path, find, repl, occ):
    src = open(SRC).read()
    assert src.count(find) >= occ + 1, "plant target not found: %r" % find
    parts = src.split(find)
    out = find.join(parts[:occ + 1]) + repl + find.join(parts[occ + 1:])
    assert out != src
    cfile = tmp_path / "planted.c"
    cfile.write_text(out)
    so = str(tmp_path / "libplanted.so")
    subprocess.run(["gcc", "-O1", "-fopenmp", "-fPIC", "-shared", "-std=c11", "-o", so,
                    str(cfile), "-lm"], check=True)
    return orc.load(so)


@pytest.mark.parametrize("name,find,repl,occ", PLANTS, ids=[p[0] for p in PLANTS])
def test_plant_is_caught(tmp_path, name, find, repl, occ):
    lib = _planted_lib(tmp_path, find, repl, occ)
    caught = []
    for pin in pins.ALL_PINS:
        try:
            pin(lib)
        except (AssertionError, ValueError):
            caught.append(pin.__name__)
    assert caught, "planted mistake %r passed every pin" % name
