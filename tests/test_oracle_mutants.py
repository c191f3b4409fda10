"""Mutation test of the oracle's pins.

Each mutant is a copy of ``oracle/eao.c`` with one plausible mistake planted
in it (a dropped term, a wrong sign, index, constant or comparison, a
transposed operand, an operand swapped for its neighbour).  The copy is
compiled with the oracle's own flags and the CPU pins run against it in a
child process (``EAO_LIB``); every mutant must make at least one pin fail.
An unmodified copy built the same way must pass, so that a failure is the
mistake's and not the mechanism's.  Mistakes that leave what the paper fixes
unchanged (a draw taken as 1-u, a layout changed in both the packer and the
unpacker) are not mutants: only GPU parity can see those conventions.
"""
import concurrent.futures as cf
import os
import subprocess
import sys


HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
PINS = ["test_oracle_pins.py", "test_oracle_sparse_pins.py", "test_oracle_scale_pins.py"]

# (name, text in eao.c, replacement, occurrences replaced)
MUTANTS = [
    # Philox4x32-10 and the draws
    ("philox multiplier", "M1 = 0xCD9E8D57u", "M1 = 0xCD9E8D55u", 1),
    ("philox key bumped before the first round", "if (r > 0) { k0 += W0; k1 += W1; }",
     "{ k0 += W0; k1 += W1; }", 1),
    ("philox output words swapped", "c0 = n0; c1 = lo1; c2 = n2; c3 = lo0;", "c0 = n0; c1 = lo0; c2 = n2; c3 = lo1;", 1),
    ("draw counter: t and stream swapped", "(uint32_t)(j >> 32), t, stream }", "(uint32_t)(j >> 32), stream, t }", 1),
    ("draw takes the next output word", "u[i] = (float)(r[n & 3] >> 8)", "u[i] = (float)(r[(n + 1) & 3] >> 8)", 1),
    ("every worker draws stream 0", "eao_uniforms(c->seed, t, (uint32_t)i, n0, len, u)",
     "eao_uniforms(c->seed, t, 0u, n0, len, u)", 1),
    # message sizes and layout
    ("message words without the ragged chunk", "return ((len + 255) / 256) * 4 * b;", "return (len / 256 + 1) * 4 * b;", 1),
    ("Example 2 without the zero code", "int32_t mags = kmax - kmin + 2;", "int32_t mags = kmax - kmin + 1;", 1),
    # bucket scales
    ("scaled sign: sum instead of mean", "return (float)(sum_abs(p, n) / (double)n);", "return (float)(sum_abs(p, n));", 1),
    ("L2 norm without the square root", "sqrtf((float)sum_sq(p, n))", "((float)sum_sq(p, n))", 1),
    ("max-norm and L2 swapped", "q->scale == EAO_SCALE_MAX ? max_abs(p, n)", "q->scale != EAO_SCALE_MAX ? max_abs(p, n)", 1),
    ("norm summed in binary32", "for (int64_t j = 0; j < n; ++j) s += (double)p[j] * (double)p[j];",
     "for (int64_t j = 0; j < n; ++j) s = (float)(s + (float)(p[j] * p[j]));", 1),
    ("no pre-scale of subnormal scales", "return s < 0x1p-126f ? 0x1p64f : 1.0f;", "return 1.0f;", 1),
    # quantizers
    ("scaled sign sends zero as negative", "code[j] = p[j] < 0.0f ? 1u : 0u;", "code[j] = p[j] <= 0.0f ? 1u : 0u;", 1),
    ("scaled sign flips the sign", "deq[j] = code[j] ? -s : s;", "deq[j] = code[j] ? s : -s;", 1),
    ("stochastic rounding direction", "(u[j] < fr ? 1u : 0u)", "(u[j] > fr ? 1u : 0u)", 1),
    ("stochastic grid of 2^b + 1 levels", "const uint32_t L = (1u << q->bits) - 1u;\n    if (!(s > 0.0f)",
     "const uint32_t L = (1u << q->bits);\n    if (!(s > 0.0f)", 1),
    ("uniform level off by one", "return (float)(2 * (int32_t)c - (int32_t)L) / (float)L;",
     "return (float)(2 * (int32_t)c - (int32_t)L + 1) / (float)L;", 1),
    ("Example 1 ties away from zero", "if (a - (float)i > 0.5f) i += 1;", "if (a - (float)i >= 0.5f) i += 1;", 1),
    ("Example 1 grid of 2^k levels", "const int32_t L = (1 << k) - 1;", "const int32_t L = (1 << k);", 1),
    ("Example 1 without the clamp to 1", "if (a > (float)L) a = (float)L;", ";", 1),
    ("Example 2 rounding threshold", "(frac > 0x400000u ? 1 : 0)", "(frac >= 0x400000u ? 1 : 0)", 1),
    ("Example 2 without the clamp at 2^kmax", "if (e > kmax) e = kmax;", ";", 1),
    # Definition 3 sparsifiers
    ("top-k keeps the smallest", "if (x->key != y->key) return x->key > y->key ? -1 : 1;",
     "if (x->key != y->key) return x->key < y->key ? -1 : 1;", 1),
    ("top-k ties to the higher index", "return x->idx < y->idx ? -1 : (x->idx > y->idx ? 1 : 0);",
     "return x->idx > y->idx ? -1 : (x->idx < y->idx ? 1 : 0);", 1),
    ("top-k key keeps the sign bit", "return b & 0x7FFFFFFFu;", "return b;", 1),
    ("sparse values in reverse slot order", "deq[b0 + j] = code[b0 + j] ? scales[bi * q->keep + slot++] : 0.0f;",
     "deq[b0 + j] = code[b0 + j] ? scales[bi * q->keep + (q->keep - 1 - slot++)] : 0.0f;", 1),
    # Adam (Algorithm 2)
    ("first moment decays with beta2", "*m = beta1 * *m + omb1 * g;", "*m = beta2 * *m + omb2 * g;", 1),
    ("second moment of g, not g^2", "*v = beta2 * *v + omb2 * (g * g);", "*v = beta2 * *v + omb2 * fabsf(g);", 1),
    ("eps added to the denominator", "return lr * (m / sqrtf(v));", "return lr * (m / (sqrtf(v) + 1e-8f));", 1),
    # the round (Algorithms 1-2)
    ("worker residual sign", "ei[n] = c->qw.error_feedback ? p[n] - deq[n] : 0.0f;",
     "ei[n] = c->qw.error_feedback ? deq[n] - p[n] : 0.0f;", 1),
    ("worker residual not added", "else {\n            for (int64_t n = 0; n < len; ++n) p[n] = gi[n] + ei[n];",
     "else {\n            for (int64_t n = 0; n < len; ++n) p[n] = gi[n];", 1),
    ("sum, not average, of the workers", "const float avg = acc[n] / (float)N;", "const float avg = acc[n];", 1),
    ("server residual not added", "p[n] = a + e_s[n];", "p[n] = a;", 1),
    ("server residual sign", "e_s[n] = c->qs.error_feedback ? p[n] - deq[n] : 0.0f;",
     "e_s[n] = c->qs.error_feedback ? deq[n] - p[n] : 0.0f;", 1),
    ("apply adds the update", "x[n] = x[n] - deq[n];", "x[n] = x[n] + deq[n];", 1),
    # Section V-A toy gradient and the schedules
    ("toy gradient without the factor 2", "g[(int64_t)i * d + j] = (float)(2.0 * s);", "g[(int64_t)i * d + j] = (float)s;", 1),
    ("toy gradient with A, not its transpose", "s += (double)A[k * d + j] * res[k];", "s += (double)A[j * d + k] * res[k];", 2),
    ("toy gradient without the noise", "res[k] = ax[k] - (double)x_star[k] - (double)xi[(int64_t)i * d + k];",
     "res[k] = ax[k] - (double)x_star[k];", 1),
    ("Assumption 2 step without the square root", "*lr = s->alpha / sqrtf(Tf);", "*lr = s->alpha / Tf;", 1),
    ("step decay one step early", "int64_t k = (t - 1) / s->period;\n        float r = 1.0f, b = s->factor;\n        while",
     "int64_t k = t / s->period;\n        float r = 1.0f, b = s->factor;\n        while", 1),
]


def _source():
    with open(os.path.join(ROOT, "oracle", "eao.c")) as f:
        return f.read()


def _compile(src_text, out_dir):
    sys.path.insert(0, ROOT)
    from oracle.build import CFLAGS
    os.makedirs(out_dir, exist_ok=True)
    src = os.path.join(out_dir, "eao.c")
    with open(src, "w") as f:
        f.write(src_text)
    lib = os.path.join(out_dir, "liboracle.so")
    flags = [f for f in CFLAGS if f not in ("-Wall", "-Wextra")]
    r = subprocess.run(["gcc", *flags, "-I", os.path.join(ROOT, "oracle"), src, "-lm", "-o", lib],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-2000:]
    return lib


def _run_pins(lib):
    env = dict(os.environ)
    env["EAO_LIB"] = lib
    env["OMP_NUM_THREADS"] = "1"
    r = subprocess.run([sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider", "-m", "not gpu",
                        *[os.path.join(HERE, p) for p in PINS]], cwd=ROOT, env=env, capture_output=True,
                       text=True, timeout=600)
    return r.returncode, r.stdout[-1500:] + r.stderr[-1500:]


def test_every_mutant_fails_a_pin(tmp_path):
    src = _source()
    names = [m[0] for m in MUTANTS]
    assert len(set(names)) == len(names)
    libs = {"control": _compile(src, str(tmp_path / "control"))}
    for i, (name, old, new, count) in enumerate(MUTANTS):
        assert src.count(old) == count, f"mutant '{name}': its text occurs {src.count(old)} times in eao.c"
        libs[name] = _compile(src.replace(old, new), str(tmp_path / f"m{i}"))
    with cf.ThreadPoolExecutor(max_workers=6) as pool:
        results = dict(zip(libs, pool.map(_run_pins, libs.values())))
    rc, out = results.pop("control")
    assert rc == 0, f"the unmodified copy fails its pins:\n{out}"
    survivors = [name for name, (rc, _) in results.items() if rc == 0]
    assert not survivors, "mutants that pass every pin: " + ", ".join(survivors)
    for name, (rc, out) in results.items():
        # a kill is a failed pin (exit status 1), not a crash or a collection error
        assert rc == 1, f"mutant '{name}' ended with status {rc}:\n{out}"
