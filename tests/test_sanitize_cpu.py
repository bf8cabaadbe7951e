"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only).

Two drivers in tests/sanitize/ are built with g++ / gcc (no device code):
  - plan_driver: the library's structure reader, compiler (normal form and
    fusion) and batch lowering, fed random structures, every built-in, and
    malformed texts (truncations, substitutions, over-deep nesting, too many
    subqueries, huge slots), then random node arrays;
  - oracle_driver: the CPU oracle for all five models on random small
    parameters of exact shapes, every built-in structure with valid and
    out-of-range ids, the same graphs as node arrays (malformed ones
    included), top-k and filtered ranks with invalid arguments.
The sanitizers abort on the first error, so a clean exit means none was
found on these inputs.
"""

import os
import shutil
import subprocess

import numpy as np
import pytest

from paper_2503_02172_amd import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-g", "-O1"]

pytestmark = pytest.mark.skipif(shutil.which("g++") is None or shutil.which("gcc") is None,
                                reason="needs the host compilers g++ and gcc")


def _texts():
    """Structure texts: random ones, the built-ins, and malformed variants."""
    out = []
    for seed in range(120):
        out.append(synth.random_structure(seed, negation=bool(seed % 2)))
    out += list(synth.STRUCTURE_TEXT.values())
    rng = np.random.default_rng(5)
    good = list(out)
    for t in good[:40]:
        out += [t[:k] for k in range(0, len(t), max(1, len(t) // 6))]       # truncations
        s = list(t)
        for _ in range(3):
            s[int(rng.integers(len(s)))] = "eprinu(),0123456789x "[int(rng.integers(21))]
        out.append("".join(s))                                              # substitutions
    deep = "e0"
    for h in range(70):
        deep = f"p({deep},r{h % 8})"
    out += [deep, "i(" + ",".join(f"p(e{j},r{j})" for j in range(5)) + ")",   # too deep, 5 subqueries
            "p(e99999999999,r0)", "p(e0,r4294967296)", "u(p(e0,r0))", "n()", "", "(", "p(e0,r0))",
            "i(p(e0,r0),e1)", "p(n(e0),r0)", "u(n(p(e0,r0)),n(p(e1,r1)),n(p(e2,r2)),n(p(e3,r3)))",
            "i(u(p(e0,r0),p(e1,r1)),u(p(e2,r2),p(e3,r3)),u(p(e4,r4),p(e5,r5)))"]
    return out


def _build(tmp, out, srcs, cxx):
    cmd = [cxx] + SAN + (["-std=c++17"] if cxx == "g++" else ["-std=gnu11", "-fopenmp"]) + srcs + ["-o", out]
    if cxx == "gcc":
        cmd += ["-lm"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-3000:]


def _run(cmd):
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:abort_on_error=1", UBSAN_OPTIONS="print_stacktrace=1",
               OMP_NUM_THREADS="2")
    r = subprocess.run(cmd, capture_output=True, text=True, env=env, timeout=600)
    bad = ("ERROR: AddressSanitizer" in r.stderr) or ("runtime error" in r.stderr)
    assert r.returncode == 0 and not bad, (r.returncode, r.stderr[-4000:])
    return r.stdout


def test_plan_compiler_under_sanitizers(tmp_path):
    exe = str(tmp_path / "plan_driver")
    _build(tmp_path, exe, [os.path.join(ROOT, "tests", "sanitize", "plan_driver.cpp"),
                           os.path.join(ROOT, "paper_2503_02172_amd", "csrc", "plan.cpp")], "g++")
    texts = tmp_path / "texts.txt"
    texts.write_text("\n".join(_texts()) + "\n")
    out = _run([exe, str(texts), "11"])
    counts = dict(zip(out.split()[::2], out.split()[1::2]))
    print(out)
    assert int(counts["parsed"]) >= 130 and int(counts["compiled"]) > 0 and int(counts["lowered"]) > 0


def test_oracle_under_sanitizers(tmp_path):
    exe = str(tmp_path / "oracle_driver")
    _build(tmp_path, exe, [os.path.join(ROOT, "tests", "sanitize", "oracle_driver.c")], "gcc")
    lines = []
    for t in _texts():
        try:
            g = synth.graph_nodes(t)
        except (ValueError, IndexError, RecursionError, OverflowError):
            continue
        lines.append(" ".join([str(g.shape[0])] + [str(int(v)) for v in g.reshape(-1)]))
    rng = np.random.default_rng(6)
    for _ in range(60):                       # malformed node arrays
        n = int(rng.integers(1, 12))
        g = np.stack([rng.integers(-1, 6, n), rng.integers(-2, 10, n)] +
                     [rng.integers(-2, n + 2, n) for _ in range(4)], 1)
        lines.append(" ".join([str(n)] + [str(int(v)) for v in g.reshape(-1)]))
    graphs = tmp_path / "graphs.txt"
    graphs.write_text("\n".join(lines) + "\n")
    out = _run([exe, str(graphs), "12"])
    print(out)
    assert int(out.split()[1]) > 0


def test_sanitizers_catch_a_planted_overflow(tmp_path):
    """The same flags on a program with a heap read one past the end: the run
    must fail with a sanitizer report, so a clean run above means something."""
    src = tmp_path / "planted.c"
    src.write_text("#include <stdlib.h>\nint main(int c, char** v) { int* p = malloc(4 * sizeof(int));\n"
                   "  p[0] = c; volatile int x = p[4 + (c > 5)]; free(p); return x == 12345; }\n")
    exe = str(tmp_path / "planted")
    r = subprocess.run(["gcc"] + SAN + [str(src), "-o", exe], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    r = subprocess.run([exe], capture_output=True, text=True,
                       env=dict(os.environ, ASAN_OPTIONS="detect_leaks=0"))
    assert r.returncode != 0 and ("heap-buffer-overflow" in r.stderr or "runtime error" in r.stderr)
