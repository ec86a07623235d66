"""Planted-mistake check of the oracle's pins (CPU only; run by hand:
``python tests/oracle_mutants.py [NAME ...]``).

Each mutant is oracle/oracle.c with one plausible mistake: a wrong rounding
tie rule or threshold in the FP16 conversion, a wrong sign or a missing scale
in the split, a dropped or swapped term or a misread parenthesisation in one
of the accumulation orders (Sec. 4.5), a dropped k.  Each is built into a
temporary directory and the oracle's tests run against it (through
SGEMM_CUBE_ORACLE_LIB); the built oracle/liboracle.so is never touched.  A
mutant the tests do not reject would be a gap in the pins, so every one must
be killed."""
import os
import subprocess
import sys
import tempfile

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "oracle.c")
# The fast tests first: a run stops at the first failure.
TESTS = ["tests/test_oracle_folds.py", "tests/test_oracle_gemm.py", "tests/test_oracle_split.py",
         "tests/test_bounds.py", "tests/test_parity_bar.py", "tests/test_oracle_range.py",
         "tests/test_oracle_convert.py"]
MUTANTS = {
    "normal ties away from zero": (
        "(rest == 0x1000u && (keep & 1u))", "(rest == 0x1000u)"),
    "overflow threshold at 65504": (
        "if (ax >= 0x477ff000u)", "if (ax >= 0x477fe000u)"),
    "flush below 2^-24": (
        "if (ax < 0x33000000u)", "if (ax < 0x33800000u)"),
    "subnormal ties away": (
        "if (rem > half || (rem == half && (q & 1u))) q += 1u;", "if (rem >= half) q += 1u;"),
    "NaN with payload 1 to inf": (
        "if (ax > 0x7f800000u) /* NaN */", "if (ax > 0x7f800001u) /* NaN */"),
    "subnormal widening off by a factor 2": (
        "(float)m * 0x1p-24f", "(float)m * 0x1p-25f"),
    "residual sign flipped": (
        "float r = a - widen(h);", "float r = widen(h) - a;"),
    "lo not scaled": (
        "float rs = r * scale;", "float rs = r;"),
    "last k dropped": (
        "for (int64_t k = k0; k < k1; ++k) {", "for (int64_t k = k0; k < k1 - (k1 == K); ++k) {"),
    "elementwise XB before XA": (
        "t = t + xa[j] * inv_s;\n                HH[j] = t + xb[j] * inv_s;",
        "t = t + xb[j] * inv_s;\n                HH[j] = t + xa[j] * inv_s;"),
    "elementwise block folded first": (
        "float t = HH[j] + hh[j];\n                t = t + xa[j] * inv_s;\n"
        "                HH[j] = t + xb[j] * inv_s;",
        "float t = hh[j] + xa[j] * inv_s;\n                t = t + xb[j] * inv_s;\n"
        "                HH[j] = HH[j] + t;"),
    "elementwise drops XB": (
        "HH[j] = t + xb[j] * inv_s;", "HH[j] = t;"),
    "termwise cross sums added first": (
        "float t = HH[j] + XA[j] * inv_s;\n            C[i * ldc + j] = t + XB[j] * inv_s;",
        "C[i * ldc + j] = HH[j] + (XA[j] + XB[j]) * inv_s;"),
    "termwise XB accumulates XA": (
        "XB[j] = XB[j] + xb[j];", "XB[j] = XB[j] + xa[j];"),
    "cross-first as (acc + HH_g) + X_g/s": (
        "float blk = cross * inv_s + hh[j];\n                HH[j] = HH[j] + blk;",
        "float blk = HH[j] + hh[j];\n                HH[j] = blk + cross * inv_s;"),
    "cross-first without XB": (
        "float cross = xa[j] + xb[j];", "float cross = xa[j];"),
}


def run_mutant(name: str, workdir: str):
    """(killed, first failing test) for one mutant."""
    before, after = MUTANTS[name]
    src = open(SRC).read()
    if src.count(before) != 1:
        raise SystemExit(f"mutant {name!r} no longer matches oracle.c")
    cfile = os.path.join(workdir, "oracle.c")
    lib = os.path.join(workdir, "liboracle.so")
    with open(cfile, "w") as f:
        f.write(src.replace(before, after))
    r = subprocess.run(["gcc", "-O3", "-std=c11", "-fPIC", "-shared", "-fopenmp",
                        "-fno-fast-math", "-ffp-contract=off", "-march=x86-64-v3", cfile,
                        "-o", lib, "-lm"], capture_output=True, text=True)
    if r.returncode != 0:
        raise SystemExit(r.stderr)
    env = dict(os.environ, SGEMM_CUBE_ORACLE_LIB=lib)
    r = subprocess.run([sys.executable, "-m", "pytest", *TESTS, "-x", "-q", "-p",
                        "no:cacheprovider"], capture_output=True, text=True, cwd=ROOT, env=env,
                       timeout=1800)
    failed = [ln for ln in r.stdout.splitlines() if ln.startswith("FAILED")]
    return r.returncode != 0, (failed[0][7:] if failed else "")


def main(names):
    survivors = []
    for name in names or list(MUTANTS):
        with tempfile.TemporaryDirectory() as d:
            killed, test = run_mutant(name, d)
        print(f"{'killed  ' if killed else 'SURVIVED'} {name}" + (f"  <- {test}" if killed else ""),
              flush=True)
        if not killed:
            survivors.append(name)
    return 1 if survivors else 0


if __name__ == "__main__":
    sys.exit(main(sys.argv[1:]))
