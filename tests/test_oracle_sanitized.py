"""The C oracle under AddressSanitizer and UndefinedBehaviorSanitizer (CPU only).

The oracle is compiled a second time with -fsanitize=address,undefined and run,
in a child process that preloads the sanitizer runtime, over the inputs most
likely to expose a memory or integer error: every valid stream up to 10 tokens
and corrupted copies of them, nesting 2000 deep, 300-entry fan-out with a
thread-count mismatch, all-tag rows, empty and truncated rows; then the group
reward (both normalisation modes) and the batch metrics.  Any sanitizer report
aborts the child; its results must also equal, bit for bit, those of the
normal build."""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "parason_oracle.c")

CHILD = r'''
import random, sys
import numpy as np
sys.path.insert(0, ROOT)
sys.path.insert(0, os.path.join(ROOT, "tests"))
from oracle import oracle as O
import grammar_pins as GP

TAGS = np.arange(100, 112, dtype=np.int32)
streams = [list(s) for s in GP.enumerate_valid(10)]
rng = random.Random(3)
for s in list(streams):
    t = list(s)
    t[rng.randrange(len(t))] = rng.randrange(13)
    streams.append(t)
    streams.append(s[: rng.randrange(len(s) + 1)])
d = 2000
streams.append([GP.THINK] + [GP.PAR, GP.OUT, GP.TRI, GP.TEXT, GP.END_TRI, GP.END_OUT, GP.THR, GP.TEXT] * d
               + [GP.END_THR, GP.END_PAR] * d + [GP.END_THINK])
fan = [GP.THINK, GP.PAR, GP.OUT] + [GP.SUB, GP.TEXT, GP.END_SUB] * 300 + [GP.END_OUT]
streams.append(fan + [GP.THR, GP.END_THR] * 250 + [GP.END_PAR, GP.END_THINK])
streams.append([rng.randrange(1, 13) for _ in range(10000)])
streams += [[], [GP.TEXT], [GP.THINK]]
n = len(streams) // 8 * 8
streams = streams[:n]
toks = [GP.to_tokens(s, TAGS) for s in streams]
lengths = np.array([len(t) for t in toks], np.int32)
starts = np.zeros(n, np.int64)
starts[1:] = np.cumsum(lengths[:-1].astype(np.int64))
flat = np.array([x for t in toks for x in t] or [0], np.int32)
correct = np.array([rng.randrange(2) for _ in range(n)], np.uint8)

def run():
    rows = O.eval_rows(flat, starts, lengths, TAGS)
    out = [rows.tobytes()]
    for flags in (0, O.CFG_INVALID_KEEPS_CORRECTNESS, O.CFG_BATCH_STATS):
        R = O.group_reward(rows, correct, 8, 0.1, 0.05, 0.1, 0.5, 0.25, flags)
        out += [np.asarray(x).tobytes() for x in R]
    m = O.batch_metrics(rows, correct, O.group_reward(rows, correct, 8, 0.1, 0.0, 0.1, 0.5, 0.25)[0])
    out.append(repr(sorted(m.items())).encode())
    return out

O.LIB = SANITIZED
O._lib = None
got = run()
O.LIB = NORMAL
O._lib = None
ref = run()
assert got == ref, "sanitized and normal builds disagree"
print("ok", n, "rows")
'''


def test_oracle_under_sanitizers(tmp_path):
    gcc = shutil.which("gcc")
    if gcc is None:
        pytest.skip("gcc not available")
    asan = subprocess.run([gcc, "-print-file-name=libasan.so"], capture_output=True, text=True).stdout.strip()
    if not asan or not os.path.isabs(asan) or not os.path.exists(asan):
        pytest.skip("libasan not available")
    lib = str(tmp_path / "liboracle_san.so")
    subprocess.check_call([gcc, "-O1", "-g", "-std=c99", "-fPIC", "-shared", "-ffp-contract=off",
                           "-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer",
                           "-o", lib, SRC, "-lm", "-lpthread"])
    from oracle import oracle as O

    normal = O.build()
    script = "import os\nROOT = %r\nSANITIZED = %r\nNORMAL = %r\n" % (ROOT, lib, normal) + CHILD
    env = dict(os.environ, LD_PRELOAD=asan, ASAN_OPTIONS="detect_leaks=0:abort_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1")
    r = subprocess.run([sys.executable, "-c", script], env=env, capture_output=True, text=True, timeout=600)
    assert r.returncode == 0, (r.stdout[-2000:], r.stderr[-4000:])
    assert r.stdout.startswith("ok")
