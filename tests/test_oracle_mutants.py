"""Planted mistakes in copies of the oracle (CPU only).

The oracle's pins should fail on any plausible slip in the code they guard.
This test checks that.  Each mutant is one small edit to a copy of
oracle.c: a dropped term, a wrong sign, index, constant or comparison, or a
transposed operand.  The copy is built with the oracle's own flags, and the
oracle's pin tests run against it in a subprocess (CDT_ORACLE_LIB points the
oracle's loader at the copy).  At least one pin must fail for every mutant.
The unmodified copy must pass, which shows that the harness itself does not
fail by accident.  The mistakes are planted in the oracle only; nothing here
touches the GPU library.
"""
import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor


from tests.conftest import ROOT

SRC = os.path.join(ROOT, "oracle", "oracle.c")
PIN_FILES = ["tests/test_oracle_rng.py", "tests/test_oracle_generator.py",
             "tests/test_oracle_drift.py", "tests/test_oracle_auroc.py",
             "tests/test_oracle_ablations.py", "tests/test_oracle_outcomes.py"]

# (name, text in oracle.c, replacement)
MUTANTS = [
    # Philox4x32-10 (Salmon et al., SC'11)
    ("philox multiplier", "PHILOX_MUL0 = 0xD2511F53u", "PHILOX_MUL0 = 0xD2511F57u"),
    ("philox round count", "round < 10; ++round", "round < 9; ++round"),
    ("philox transposed product", "uint32_t y0 = (uint32_t)(p1 >> 32) ^ x1 ^ k0;",
     "uint32_t y0 = (uint32_t)(p0 >> 32) ^ x1 ^ k0;"),
    ("philox key increment", "k1 += PHILOX_WEYL1;", "k1 += PHILOX_WEYL0;"),
    # Irwin-Hall normal and fp16 rounding
    ("irwin-hall centre", "(int32_t)(w1 >> 16) - 131070;", "(int32_t)(w1 >> 16) - 131072;"),
    ("irwin-hall scale", "sqrt(3.0 / 4294967295.0)", "sqrt(1.0 / 4294967295.0)"),
    ("f16 ties away from zero", "(frac == 0.5 && fmod(f, 2.0) == 1.0)", "(frac == 0.5)"),
    ("f16 overflow check missing", "if (ax >= 65520.0)\n        return (uint16_t)(sign | 0x7C00u);",
     "if (0)\n        return (uint16_t)(sign | 0x7C00u);"),
    ("f16 subnormal spacing", "quantum = 0x1p-24; /* subnormal spacing */",
     "quantum = 0x1p-25; /* subnormal spacing */"),
    ("f16 value subnormal", "return sign * ldexp((double)mant, -24);",
     "return sign * ldexp((double)mant, -25);"),
    # synthetic references and block statistics
    ("reference gain dropped", "out[k] = r32((double)z * (double)gain[j]);",
     "out[k] = r32((double)z);"),
    ("reference channel index", "uint32_t j = e % H;", "uint32_t j = (e / H) % H;"),
    ("outlier order reversed", "return a->word < b->word ? -1 : 1;",
     "return a->word > b->word ? -1 : 1;"),
    ("mean |a| without abs", "m += fabs(x);", "m += x;"),
    ("rms without sqrt", "double rms = n > 0 ? sqrt(sumsq[b] / n) : 0.0;",
     "double rms = n > 0 ? sumsq[b] / n : 0.0;"),
    ("block scale from rms", "double mu = n > 0 ? sumabs[b] / n : 0.0;",
     "double mu = n > 0 ? sqrt(sumsq[b] / n) : 0.0;"),
    # live pass (Eqs. 2-3)
    ("benign scale sign", "r32((double)sigma_f * fabs((double)a))",
     "r32((double)sigma_f * (double)a)"),
    ("benign counter transposed", "float zb = normal1(seed, st_benign, cfg_id, s, c, e);",
     "float zb = normal1(seed, st_benign, cfg_id, c, s, e);"),
    ("student-t third term", "(double)r32((double)z3 * z3));", "0.0);"),
    ("tamper ignores benign output",
     "v = r32((double)v + (double)r32((double)tscale * (double)zt));",
     "v = r32((double)base + (double)r32((double)tscale * (double)zt));"),
    ("flip selects complement", "return (double)u < thr;", "return (double)u > thr;"),
    ("carry sign", "return (s == 0) ? a : r32((double)a + (double)r32((double)g * (double)d));",
     "return (s == 0) ? a : r32((double)a - (double)r32((double)g * (double)d));"),
    ("carry from reference", "d = r32(orc_f16_value(hb) - (double)a);",
     "d = r32(orc_f16_value(hb) - (double)u);"),
    ("exact norm without sqrt", "return zz > 0.0 ? r32(eps * sqrt(vv / zz)) : 0.0f;",
     "return zz > 0.0 ? r32(eps * vv / zz) : 0.0f;"),
    ("exact norm of reference", "vv += (double)v * (double)v;", "vv += (double)a * (double)a;"),
    ("chain exact norm drops earlier tampers", "tscale[b], flip_p, scale_f, u, v);",
     "0.0f, flip_p, scale_f, u, v);"),
    ("chain exact norm of the reference", "float vt = (tamper_base == ORC_BASE_CLEAN) ? u : v;",
     "float vt = a;"),
    # Eq. 4 and its ablations
    ("drift denominator from h", "        R += av * av;\n", "        R += hv * hv;\n"),
    ("drift without sqrt", "        return D == 0.0 ? 0.0 : INFINITY;\n    return sqrt(D / R);\n}\n\n/* Scores",
     "        return D == 0.0 ? 0.0 : INFINITY;\n    return D / R;\n}\n\n/* Scores"),
    ("drift degenerate block", "        return D == 0.0 ? 0.0 : INFINITY;\n    return sqrt(D / R);\n}\n\n/* Scores",
     "        return 0.0;\n    return sqrt(D / R);\n}\n\n/* Scores"),
    ("score layout transposed",
     "double m = orc_drift_block(n, h + b * n, ref + b * n, &D, &R);\n            uint64_t o = (uint64_t)c * S + s;",
     "double m = orc_drift_block(n, h + b * n, ref + b * n, &D, &R);\n            uint64_t o = (uint64_t)s * C + c;"),
    ("cosine sign", "return (double)(1.0L - ha / sqrtl(hh * aa));",
     "return (double)(1.0L + ha / sqrtl(hh * aa));"),
    # Eqs. 5-6, control and random baseline
    ("ties counted as wins", "counts[0] += (r > 0);", "counts[0] += (r >= 0);"),
    ("NaN ranked lowest", "return nx && ny ? 0 : (nx ? 1 : -1);",
     "return nx && ny ? 0 : (nx ? -1 : 1);"),
    ("control keeps true positives",
     "if (!(flags & ORC_CTRL_INCLUDE_TRUE) && ((pos_mask >> j) & 1u))",
     "if ((flags & ORC_CTRL_INCLUDE_TRUE) && ((pos_mask >> j) & 1u))"),
    ("random score bits", "(double)(w[0] >> 8) * 0x1p-24", "(double)(w[0] >> 9) * 0x1p-24"),
    ("pooled order reversed", "pooled[0] += (r > 0);", "pooled[0] += (r < 0);"),
    # Eq. 5 per canary
    ("per-canary ties as wins", "o[0] += (r > 0);", "o[0] += (r >= 0);"),
    ("per-canary draws at the local index", "const uint32_t tg = canary_base + t;",
     "const uint32_t tg = t;"),
    ("per-canary control keeps true positives", "if (skip_true && ((pos_mask >> j) & 1u))",
     "if (!skip_true && ((pos_mask >> j) & 1u))"),
    ("per-canary baseline compares a stage with itself",
     "int q = score_cmp(orc_random_score(seed, cfg_id, tg, i),",
     "int q = score_cmp(orc_random_score(seed, cfg_id, tg, j),"),
]

CFLAGS = ["-O2", "-std=c11", "-fPIC", "-shared", "-ffp-contract=off", "-fno-fast-math"]


def _build(text, out):
    subprocess.run(["gcc", *CFLAGS, "-x", "c", "-", "-o", out, "-lm"], input=text.encode(),
                   check=True, capture_output=True)


def _pins_fail(lib):
    env = dict(os.environ, CDT_ORACLE_LIB=lib)
    env.pop("CDT_SLOW", None)
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider",
                        *PIN_FILES], cwd=ROOT, env=env, capture_output=True, text=True,
                       timeout=600)
    return r.returncode != 0, r.stdout[-2000:]


def test_mutant_texts_are_unique():
    src = open(SRC).read()
    for name, old, new in MUTANTS:
        assert src.count(old) == 1, f"{name}: the planted text must occur exactly once"
        assert old != new, name


def test_every_planted_mistake_fails_a_pin(tmp_path):
    src = open(SRC).read()
    jobs = [("unmodified", src)]
    for name, old, new in MUTANTS:
        jobs.append((name, src.replace(old, new)))
    libs = []
    for k, (name, text) in enumerate(jobs):
        lib = str(tmp_path / f"liboracle_{k}.so")
        _build(text, lib)
        libs.append(lib)
    with ThreadPoolExecutor(max_workers=max(1, min(6, (os.cpu_count() or 2) - 1))) as ex:
        results = list(ex.map(_pins_fail, libs))
    failed0, out0 = results[0]
    assert not failed0, "the unmodified copy must pass its pins:\n" + out0
    survivors = [name for (name, _), (failed, _) in zip(jobs[1:], results[1:]) if not failed]
    assert not survivors, f"planted mistakes no pin catches: {survivors}"
