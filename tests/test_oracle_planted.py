"""Planted mistakes in the oracle, on the CPU: each plausible mistake below
is written into a copy of oracle/uq_oracle.c, the copy is built with the
oracle's own flags, and every CPU pin of the oracle (PIN_FILES) runs
against it in a subprocess (UQ_ORACLE_LIB).  Every mistake must make at
least one pin fail, and the unchanged copy must pass them all, so the pins
are shown to pin the oracle and not only to agree with it."""
import os
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

import pytest

from oracle import build as oracle_build

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))

# name -> [(text in uq_oracle.c, replacement)]; each text occurs exactly once
MISTAKES = {
    "butterfly sign": [("p[i + h] = a - b;", "p[i + h] = b - a;")],
    "rotation not normalised": [("for (int i = 0; i < d; ++i) p[i] = p[i] * inv_sqrt;", "")],
    "exponent floored, not rounded": [("int E = (e - 1) + ((2.0 * f >= sqrt(2.0)) ? 1 : 0);", "int E = (e - 1);")],
    "E2M1 ties to the odd code": [("fabs(a - kE2M1Mag[k]);\n        if (d < best_d || (d == best_d && (k % 2) == 0))",
                                   "fabs(a - kE2M1Mag[k]);\n        if (d < best_d || (d == best_d && (k % 2) == 1))")],
    "E4M3 ties to the odd code": [("fabs(a - uqo_e4m3_value((uint8_t)k));\n        if (d < best_d || (d == best_d && (k % 2) == 0))",
                                   "fabs(a - uqo_e4m3_value((uint8_t)k));\n        if (d < best_d || (d == best_d && (k % 2) == 1))")],
    "sign bit dropped": [("return (uint8_t)((signbit(x) ? 8 : 0) | best);", "return (uint8_t)best;")],
    "nibbles swapped": [("if (ch % 2 == 0) ct[off]", "if (ch % 2 == 1) ct[off]"),
                        ("codes[ch] = (ch % 2 == 0) ? (b & 0x0F) : (b >> 4);",
                         "codes[ch] = (ch % 2 == 1) ? (b & 0x0F) : (b >> 4);")],
    "K tile token-major": [("if (kv == 0) return ((ch / 32) * 16 + t) * 16 + (ch % 32) / 2;",
                            "if (kv == 0) return (t * (d / 32) + ch / 32) * 16 + (ch % 32) / 2;")],
    "GQA map interleaved": [("const int hk = hq / G;\n            const int ctx = context_lens[b];",
                             "const int hk = hq % num_kv_heads;\n            const int ctx = context_lens[b];")],
    "softmax scale dropped": [("s[j] = softmax_scale * dot;", "s[j] = dot;")],
    "output not rotated back": [("if (rotate_v) uqo_wht_f64(acc, o, d);", "if (0) uqo_wht_f64(acc, o, d);")],
    "TQ4 key norm not square-rooted": [("return (float)sqrtq(s);", "return (float)s;")],
    "TQ4 key norm from fp32 squares": [("s += (__float128)x[c] * (__float128)x[c];", "s += (__float128)(x[c] * x[c]);")],
    "TQ4 key index ties to the upper level": [("idx += (__float128)x > mid[j] * (__float128)n;",
                                               "idx += (__float128)x >= mid[j] * (__float128)n;")],
    "TQ4 value zero point not BF16": [("const float z = uqo_bf16_rne(mn);", "const float z = mn;")],
    "TQ4 value grid of 16 steps": [("const float s = uqo_bf16_rne(d / 15.0f);", "const float s = uqo_bf16_rne(d / 16.0f);")],
    "TQ4 V tokens reversed in a dword": [("4 * (t % 4) + (c % 8) / 2; }", "4 * (3 - t % 4) + (c % 8) / 2; }")],
}
# every CPU pin of the oracle
PIN_FILES = ["test_oracle_pins.py", "test_oracle_headdim.py", "test_tq4_oracle.py", "test_calibration_cpu.py"]


def run_pins(src_text, workdir, name):
    """Build `src_text` as an oracle library and run the pins against it;
    returns pytest's exit status and the tail of its output."""
    d = os.path.join(workdir, name.replace(" ", "_").replace(",", ""))
    os.makedirs(d)
    src = os.path.join(d, "uq_oracle.c")
    with open(src, "w") as f:
        f.write(src_text)
    lib = oracle_build.build(src=src, lib=os.path.join(d, "liboracle.so"))
    env = dict(os.environ, UQ_ORACLE_LIB=lib, OMP_NUM_THREADS="2")
    r = subprocess.run([sys.executable, "-m", "pytest", "-x", "-q", "-p", "no:cacheprovider"] +
                       [os.path.join(ROOT, "tests", f) for f in PIN_FILES],
                       cwd=ROOT, env=env, capture_output=True, text=True, timeout=600)
    return r.returncode, (r.stdout + r.stderr)[-600:]


def test_every_planted_mistake_fails_a_pin(tmp_path):
    with open(oracle_build.SRC) as f:
        original = f.read()
    cases = {"unchanged": original}
    for name, edits in MISTAKES.items():
        text = original
        for old, new in edits:
            assert text.count(old) == 1, (name, old)
            text = text.replace(old, new)
        cases[name] = text
    with ThreadPoolExecutor(max_workers=4) as pool:
        results = dict(zip(cases, pool.map(lambda kv: run_pins(kv[1], str(tmp_path), kv[0]), cases.items())))
    rc, out = results.pop("unchanged")
    assert rc == 0, f"the unchanged copy fails the pins:\n{out}"
    survivors = {name: out for name, (rc, out) in results.items() if rc != 1}
    assert not survivors, "mistakes no pin caught (or that broke the run):\n" + "\n".join(
        f"--- {name}\n{out}" for name, out in survivors.items())
