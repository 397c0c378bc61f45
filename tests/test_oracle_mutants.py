"""Mutation check of the oracle's pins (CPU only).

Each mutant below is the oracle with one plausible mistake planted in a copy
of its source: a wrong index, a dropped or sign-flipped term, swapped
operands, a rounding done twice, an off-by-one in a bound.  Every mutant is
compiled on its own and the oracle's pin tests (tests/test_oracle_*.py) are
run against it; the check fails if any mutant passes them all, i.e. if the
pins would not have noticed that mistake.  The oracle's own source is never
modified."""

import concurrent.futures
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "dedloc_oracle.c")
_WORKERS = max(1, min(6, (os.cpu_count() or 2) - 1))

# pytest -k expression that leaves out the tests built on a float64
# restatement of the LAMB formula
NO_FLOAT64 = "not float64"

# (name, text in the oracle, replacement[, -k expression selecting the pins
# that must catch it])
MUTANTS = [
    ("partition: share of the wrong peer", "cum += beta ? beta[k - 1] : 1u;", "cum += beta ? beta[k] : 1u;"),
    ("weights: reciprocal instead of division", "w[p] = (float)counts[p] / (float)W;",
     "w[p] = (float)counts[p] * (1.0f / (float)W);"),
    ("fp16: ties away from zero", "if (rem > half || (rem == half && (q & 1))) q++;", "if (rem >= half) q++;"),
    ("fp16: subnormal shift off by one", "uint64_t r = shift_rne(sig, -e - 1);", "uint64_t r = shift_rne(sig, -e);"),
    ("fp16: overflow saturates instead of reaching infinity", "if (e > 15) return (uint16_t)(sign | 0x7c00u);",
     "if (e > 15) return (uint16_t)(sign | 0x7bffu);"),
    ("fp16 decode: subnormal scale", "if (e5 == 0) return s * ldexpf((float)m10, -24);",
     "if (e5 == 0) return s * ldexpf((float)m10, -25);"),
    ("fp16 decode: exponent bias", "return s * ldexpf((float)(m10 | 0x400u), (int)e5 - 25);",
     "return s * ldexpf((float)(m10 | 0x400u), (int)e5 - 24);"),
    ("fp16: NaN encoded as infinity", "if (e8 == 0xff) return (uint16_t)(sign | (m23 ? 0x7e00u : 0x7c00u));",
     "if (e8 == 0xff) return (uint16_t)(sign | 0x7c00u);"),
    ("int8: scale over 128", "float s = a / 127.0f;", "float s = a / 128.0f;"),
    ("int8: negative clamp at -128", "if (q < -127.0f) q = -127.0f;", "if (q < -128.0f) q = -128.0f;"),
    ("int8: truncation instead of rounding", "q = rintf(x[i] / s);", "q = truncf(x[i] / s);"),
    ("int8: clamp at 126", "if (q > 127.0f) q = 127.0f;", "if (q > 126.0f) q = 126.0f;"),
    ("int8 decode: wrong block", "out[i] = (float)codes[i] * scales[i / block];",
     "out[i] = (float)codes[i] * scales[(i + 1) / block];"),
    ("reduce: zero-sample peers read", "if (counts[p] == 0) continue;\n        decode_any", "decode_any"),
    ("reduce: product and sum rounded separately", "acc[e] = fmaf(w[p], dec[e], acc[e]);",
     "acc[e] = w[p] * dec[e] + acc[e];"),
    ("lamb: beta2 in the first moment", "float mn = fmaf(cfg->beta1, m[e], omb1 * gg);",
     "float mn = fmaf(cfg->beta2, m[e], omb1 * gg);"),
    ("lamb: first bias correction on v", "float vh = vn / c2;", "float vh = vn / c1;"),
    ("lamb: eps inside the square root", "float ue = mh / (sqrtf(vh) + cfg->eps) + lam * x[e];",
     "float ue = mh / sqrtf(vh + cfg->eps) + lam * x[e];"),
    ("lamb: weight decay sign", "float ue = mh / (sqrtf(vh) + cfg->eps) + lam * x[e];",
     "float ue = mh / (sqrtf(vh) + cfg->eps) - lam * x[e];"),
    ("lamb: trust ratio inverted", "r = (float)(X / U);", "r = (float)(U / X);"),
    ("lamb: update sign", "x[e] = x[e] - lrr * u[e];", "x[e] = x[e] + lrr * u[e];"),
    ("lamb: decay flag read as the adapt flag", "if (!cfg->force_unit_trust && (flags[t] & 2) && X > 0.0 && U > 0.0)",
     "if (!cfg->force_unit_trust && (flags[t] & 1) && X > 0.0 && U > 0.0)"),
    ("lamb: bias correction one step behind", "c1 = (float)(1.0 - pow((double)cfg->beta1, (double)cfg->step));",
     "c1 = (float)(1.0 - pow((double)cfg->beta1, (double)(cfg->step - 1) + 1e-9));"),
    ("lamb: NaN norms pass the zero rule", "if (!cfg->force_unit_trust && (flags[t] & 2) && X > 0.0 && U > 0.0)",
     "if (!cfg->force_unit_trust && (flags[t] & 2) && X != 0.0 && U != 0.0)"),
    ("lars: NaN norms pass the zero rule", "if (!cfg->force_unit_trust && (flags[t] & 2) && X > 0.0 && G > 0.0)",
     "if (!cfg->force_unit_trust && (flags[t] & 2) && X != 0.0 && G != 0.0)"),
    ("lars: decay term on the gradient norm", "r = (float)((double)cfg->trust_coef * X / (G + (double)lam * X));",
     "r = (float)((double)cfg->trust_coef * X / (G + (double)lam * G));"),
    ("lars: decay dropped from the step", "float d = g[e] + lam * x[e];", "float d = g[e];"),
    ("lars: momentum on the step", "float vn = fmaf(cfg->momentum, v[e], s * d);",
     "float vn = fmaf(cfg->momentum, s * d, v[e]);"),
    ("round: shard offset in elements, not bytes", "pc[p] = (const char *)peer_codes[p] + b0 * cb;",
     "pc[p] = (const char *)peer_codes[p] + b0;"),
    ("group: digit stride", "const uint32_t base = (g / lo) * lo * m + (g % lo);",
     "const uint32_t base = (g / lo) * m + (g % lo);"),
    ("group: a member counted once per group", "ncnt[s] = gt;", "ncnt[s] = cnt[s];"),
    ("accumulate: batch size dropped", "acc[i] = fmaf(b, gi, acc[i]);", "acc[i] = acc[i] + gi;"),
    ("finalize: reciprocal instead of division", "scratch[i] = acc[i] / c;", "scratch[i] = acc[i] * (1.0f / c);"),
    ("finalize: reset ignored", "    if (reset)\n        for (size_t i = 0; i < n; i++) acc[i] = 0.0f;",
     "    (void)reset;"),
    ("accumulate: fp16 codes read as their integer value",
     "float gi = g_codec == 0 ? ((const float *)g)[i] : f16_to_f32(((const uint16_t *)g)[i]);",
     "float gi = g_codec == 0 ? ((const float *)g)[i] : (float)((const uint16_t *)g)[i];"),
    ("group: members weighted by their original counts", "cnt[i] = ncnt[i];", "(void)ncnt;"),
    # The trust ratio's norms.  These two run with the float64 restatements of
    # LAMB deselected, so that a pin that does not restate the formula (the
    # hand-derived closed form with weight decay) has to catch them.
    ("lamb: decay term left out of ||u||", "su += (double)u[e] * (double)u[e];",
     "su += (double)(u[e] - lam * x[e]) * (double)(u[e] - lam * x[e]);", NO_FLOAT64),
    ("lamb: ||x - lr*u|| in place of ||x||", "sx += (double)x[e] * (double)x[e];\n            su",
     "sx += (double)(x[e] - cfg->lr * u[e]) * (double)(x[e] - cfg->lr * u[e]);\n            su", NO_FLOAT64),
]


# (name, text in oracle/lp.py, replacement): the load-balancing LP, pinned by
# tests/test_oracle_lp.py
LP_SRC = os.path.join(ROOT, "oracle", "lp.py")
LP_MUTANTS = [
    ("lp: compute rate times B", "[(c(i), -s[i] / B) for i in range(n)]", "[(c(i), -s[i] * B) for i in range(n)]"),
    ("lp: receive rate from the transposed return rates", "[(g(j, i), -1.0 / P) for j in range(n)]",
     "[(g(i, j), -1.0 / P) for j in range(n)]"),
    ("lp: aggregation without the relaxation", "add([(g(i, j), 1.0), (a(k, i), -1.0), (c(k), d[i])], d[i])",
     "add([(g(i, j), 1.0), (a(k, i), -1.0)], 0.0)"),
    ("lp: download limited by the upload bandwidth",
     "add([(a(j, i), 1.0) for j in range(n) if j != i] + [(g(j, i), 1.0) for j in range(n) if j != i], d[i])",
     "add([(a(j, i), 1.0) for j in range(n) if j != i] + [(g(j, i), 1.0) for j in range(n) if j != i], u[i])"),
    ("lp: self-traffic charged to the upload",
     "add([(a(i, j), 1.0) for j in range(n) if j != i] + [(g(i, j), 1.0) for j in range(n) if j != i], u[i])",
     "add([(a(i, j), 1.0) for j in range(n)] + [(g(i, j), 1.0) for j in range(n)], u[i])"),
    ("lp: c unbounded above", "[(0, 1)] * n", "[(0, None)] * n"),
    ("lp: a peer's own share not counted in what it receives", "[(g(j, i), -1.0 / P) for j in range(n)]",
     "[(g(j, i), -1.0 / P) for j in range(n) if j != i]"),
    ("lp: reduced form without the aggregation rate bound", "add([(g(i, j), 1.0), (h(i), -1.0)], 0.0)",
     "add([(g(i, j), 1.0), (h(i), -0.5)], 0.0)"),
]


def _lp_pins_on(src_path):
    code = ("import sys, importlib.util, oracle\n"
            f"spec = importlib.util.spec_from_file_location('oracle.lp', {src_path!r})\n"
            "mod = importlib.util.module_from_spec(spec)\n"
            "spec.loader.exec_module(mod)\n"
            "sys.modules['oracle.lp'] = mod\n"
            "oracle.lp = mod\n"
            "import pytest\n"
            "sys.exit(pytest.main(['-x', '-q', '-p', 'no:cacheprovider', 'tests/test_oracle_lp.py']))\n")
    r = subprocess.run([sys.executable, "-c", code], cwd=ROOT, capture_output=True, text=True, timeout=600)
    return r.returncode


# test files that are not pins of the C oracle: this file, the comparison of
# the oracle's two builds with each other (a mutant agrees with itself), and
# the pure-Python LP and group-size modules
_NOT_C_PINS = (os.path.basename(__file__), "test_oracle_fast_build.py", "test_oracle_lp.py",
               "test_oracle_group_size.py")


def _pins_on(lib_path, kexpr=None):
    k = ['-k', kexpr] if kexpr else []
    code = ("import os, sys, oracle\n"
            f"oracle._LIB = {lib_path!r}\n"
            "import pytest, glob\n"
            "files = sorted(glob.glob('tests/test_oracle_*.py'))\n"
            f"files = [f for f in files if os.path.basename(f) not in {_NOT_C_PINS!r}]\n"
            f"sys.exit(pytest.main(['-x', '-q', '-p', 'no:cacheprovider', '-m', 'not gpu'] + {k!r} + files))\n")
    r = subprocess.run([sys.executable, "-c", code], cwd=ROOT, capture_output=True, text=True, timeout=600)
    return r.returncode


def _mutant(i, name, old, new, tmp, kexpr=None):
    src = open(SRC).read()
    assert src.count(old) == 1, f"mutation site not unique or missing: {name}"
    c = os.path.join(tmp, f"mutant_{i}.c")
    lib = os.path.join(tmp, f"liboracle_mutant_{i}.so")
    open(c, "w").write(src.replace(old, new))
    subprocess.check_call(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-ffp-contract=off", "-fno-fast-math",
                           c, "-o", lib, "-lm"])
    return name, _pins_on(lib, kexpr)


def test_pins_catch_every_mutant(tmp_path):
    assert _pins_on(os.path.join(ROOT, "oracle", "liboracle.so")) == 0  # the real oracle passes
    assert _pins_on(os.path.join(ROOT, "oracle", "liboracle.so"), NO_FLOAT64) == 0
    with concurrent.futures.ThreadPoolExecutor(max_workers=_WORKERS) as ex:
        results = list(ex.map(lambda a: _mutant(a[0], *a[1][:3], str(tmp_path), *a[1][3:]), enumerate(MUTANTS)))
    survivors = [name for name, rc in results if rc == 0]
    assert not survivors, f"mutants the pins do not catch: {survivors}"



def test_lp_pins_catch_every_mutant(tmp_path):
    assert _lp_pins_on(LP_SRC) == 0  # the real oracle passes
    src = open(LP_SRC).read()

    def run(i, name, old, new):
        assert src.count(old) == 1, f"mutation site not unique or missing: {name}"
        path = str(tmp_path / f"lp_mutant_{i}.py")
        open(path, "w").write(src.replace(old, new))
        return name, _lp_pins_on(path)

    with concurrent.futures.ThreadPoolExecutor(max_workers=_WORKERS) as ex:
        results = list(ex.map(lambda a: run(a[0], *a[1]), enumerate(LP_MUTANTS)))
    survivors = [name for name, rc in results if rc == 0]
    assert not survivors, f"LP mutants the pins do not catch: {survivors}"


if __name__ == "__main__":
    pytest.main([__file__, "-q"])
