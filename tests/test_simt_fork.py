"""Fork/join packing runs on the CPU, under AddressSanitizer and
UndefinedBehaviorSanitizer, against the oracle.

The library's own csrc/fork.hip (with csrc/parason.hip for the handle) is
compiled for the host with the SIMT emulation of tests/simt/hip/hip_runtime.h
(lanes as fibers meeting at every wave operation), and tests/simt/emu_fork.cpp
drives it through the C-ABI: a sizing call, then a call with outputs of exactly
the returned size, every buffer sized exactly and filled with a byte pattern.
The emulated device's compute-unit count sets the grids, so a few units make
every wave of the copies walk many tiles and rows; the outputs are compared
with oracle/fork_oracle.py like the GPU tests do: row status, worker offsets,
every worker record and context token, every joined row.

Planted mistakes in copies of the kernel source (a seed text one token off, a
lost carry between scan tiles, a worker span of the join one token short)
must each be caught."""
import os
import shutil
import subprocess

import numpy as np
import pytest

from fork_cases import (CONTIG, SCATTERED, hand_rows, layout, lenient_hand_rows, oracle_fork, short_rows,
                        synthetic_main_rows, worker_sequences)
from gpu_util import insert_gaps
from oracle import fork_oracle as F
from paper_2608_24658_amd import parason as PX

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2608_24658_amd", "csrc")
SIMT = os.path.join(ROOT, "tests", "simt")
CLANG = "/opt/rocm/llvm/bin/clang++"

pytestmark = pytest.mark.skipif(not os.path.exists(CLANG), reason="no host clang++ with the sanitizers")


def build(out, csrc=CSRC):
    cmd = [CLANG, "-std=c++17", "-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
           "-ffp-contract=off", "-I", SIMT, "-I", os.path.join(ROOT, "include"), "-I", csrc, "-x", "c++",
           os.path.join(csrc, "parason.hip"), os.path.join(csrc, "fork.hip"), os.path.join(SIMT, "emu_fork.cpp"),
           "-o", out]
    subprocess.check_call(cmd)
    return out


@pytest.fixture(scope="module")
def emu(tmp_path_factory):
    return build(str(tmp_path_factory.mktemp("simt_fork") / "emu_fork"))


def _run(binary, payload, tmp):
    fin = os.path.join(tmp, "emu_fork_in_%d.bin" % os.getpid())
    fout = os.path.join(tmp, "emu_fork_out_%d.bin" % os.getpid())
    with open(fin, "wb") as f:
        f.write(payload)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:halt_on_error=1:abort_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    r = subprocess.run([binary, fin, fout], env=env, capture_output=True, text=True, timeout=600)
    if r.returncode != 0:
        raise RuntimeError("emulation failed (%d):\n%s" % (r.returncode, r.stderr[-4000:]))
    b = open(fout, "rb").read()
    os.unlink(fin)
    os.unlink(fout)
    return b


def _header(mode, tags, cfg_flags, call_flags, cus, tok, st, ln):
    return (np.array([mode], np.int32).tobytes() + np.asarray(tags, np.int32).tobytes()
            + np.array([cfg_flags, call_flags], np.uint32).tobytes() + np.array([cus], np.int32).tobytes()
            + np.array([len(st), tok.size], np.int64).tobytes() + np.ascontiguousarray(tok, np.int32).tobytes()
            + np.asarray(st, np.int64).tobytes() + np.asarray(ln, np.int32).tobytes())


class Reader:
    def __init__(self, b):
        self.b, self.off = b, 0

    def take(self, dtype, n):
        a = np.frombuffer(self.b, dtype, int(n), self.off).copy()
        self.off += a.nbytes
        return a


def emu_fork(binary, tok, st, ln, tags, seed, lenient=False, cus=2, tmp="/tmp"):
    b = _run(binary, _header(0, tags, PX.CFG_LENIENT_GAPS if lenient else 0, PX.FORK_SEED_ENTRY if seed else 0, cus,
                             tok, st, ln), tmp)
    r = Reader(b)
    rc0, rc1 = r.take(np.int32, 2)
    assert rc0 == PX.OK and rc1 == PX.OK, (rc0, rc1)
    n = len(st)
    out = {"totals": r.take(np.int64, 3), "row_status": r.take(np.uint32, n), "worker_off": r.take(np.int64, n + 1)}
    W, T = int(out["totals"][0]), int(out["totals"][1])
    out["ctx_starts"] = r.take(np.int64, W)
    for k in ("ctx_lengths", "ctx_row", "ctx_entry", "ctx_kind"):
        out[k] = r.take(np.int32, W)
    out["ctx_tokens"] = r.take(np.int32, T)
    assert r.off == len(b)
    return out


def emu_join(binary, rows_layout, worker_off, seqs_layout, tags, flags, cus=2, tmp="/tmp"):
    tok, st, ln = rows_layout
    wtok, wst, wln = seqs_layout
    payload = (_header(1, tags, 0, flags, cus, tok, st, ln)
               + np.array([len(wst), wtok.size], np.int64).tobytes() + np.asarray(worker_off, np.int64).tobytes()
               + np.ascontiguousarray(wtok, np.int32).tobytes() + np.asarray(wst, np.int64).tobytes()
               + np.asarray(wln, np.int32).tobytes())
    r = Reader(_run(binary, payload, tmp))
    rc0, rc1 = r.take(np.int32, 2)
    assert rc0 == PX.OK and rc1 == PX.OK, (rc0, rc1)
    n = len(st)
    out = {"totals": r.take(np.int64, 2), "row_status": r.take(np.uint32, n), "lengths": r.take(np.int32, n),
           "starts": r.take(np.int64, n + 1)}
    out["tokens"] = r.take(np.int32, out["totals"][0])
    return out


def check_fork(binary, rows, tags, seed, rng, what, lenient=False, cus=2):
    tok, st, ln = layout(rows, rng)
    res, exp_starts, exp_lens, exp_flat = oracle_fork(rows, tags, seed, lenient)
    g = emu_fork(binary, tok, st, ln, tags, seed, lenient, cus)
    assert np.array_equal(g["row_status"], np.array(res["status"], np.uint32)), what
    assert np.array_equal(g["worker_off"], np.array(res["worker_off"], np.int64)), what
    assert list(g["totals"]) == [res["worker_off"][-1], int(exp_lens.sum()), 0], what
    assert np.array_equal(g["ctx_row"], np.array(res["row"], np.int32)), what
    assert np.array_equal(g["ctx_entry"], np.array(res["entry"], np.int32)), what
    assert np.array_equal(g["ctx_kind"], np.array([1 if k == F.SUB else 2 for k in res["kind"]], np.int32)), what
    assert np.array_equal(g["ctx_starts"], exp_starts), what
    assert np.array_equal(g["ctx_lengths"], exp_lens.astype(np.int32)), what
    if not np.array_equal(g["ctx_tokens"], exp_flat):
        bad = np.nonzero(g["ctx_tokens"] != exp_flat)[0]
        w = int(np.searchsorted(exp_starts, bad[0], side="right") - 1)
        raise AssertionError("%s: %d context tokens differ, first at %d (worker %d, row %d)" % (
            what, bad.size, bad[0], w, res["row"][w]))
    return res


def check_join(binary, rows, res, seqs, tags, rng, flags, what, cus=2):
    rl = layout(rows, rng)
    sl = layout(seqs, rng)
    exp, exp_st = F.join(rows, res["worker_off"], seqs, tags, flags=flags)
    g = emu_join(binary, rl, res["worker_off"], sl, tags, flags, cus)
    assert np.array_equal(g["row_status"], np.array(exp_st, np.uint32)), what
    lens = np.array([len(r) for r in exp], np.int64)
    assert np.array_equal(g["lengths"], lens.astype(np.int32)), what
    assert g["starts"][0] == 0 and np.array_equal(np.diff(g["starts"]), lens), what
    assert np.array_equal(g["tokens"], np.array([x for r in exp for x in r], np.int32)), what
    assert list(g["totals"]) == [int(lens.sum()), 0], what


@pytest.mark.parametrize("tags", [CONTIG, SCATTERED], ids=["contiguous", "scattered"])
@pytest.mark.parametrize("seed", [True, False], ids=["seed", "noseed"])
def test_emulated_fork_join_hand_rows(emu, tags, seed):
    rng = np.random.default_rng(1)
    rows = hand_rows(tags, [7, 8, 9, 1000, 150000])
    res = check_fork(emu, rows, tags, seed, rng, "hand")
    assert sum(s == 0 for s in res["status"]) >= 12
    seqs = worker_sequences(res, tags, rng, p_bad=0.2)
    for flags in (F.JOIN_CLOSE_PARALLEL, 0, F.JOIN_APPEND_ONLY, F.JOIN_CLOSE_PARALLEL | F.JOIN_APPEND_ONLY):
        check_join(emu, rows, res, seqs, tags, rng, flags, "hand join %d" % flags)


@pytest.mark.parametrize("workload,n,cus", [("small", 96, 1), ("small", 96, 16), ("ragged", 160, 2)])
def test_emulated_fork_join_synthetic(emu, workload, n, cus):
    rng = np.random.default_rng(2)
    rows = synthetic_main_rows(workload, n, CONTIG, seed=3)
    res = check_fork(emu, rows, CONTIG, True, rng, workload, cus=cus)
    assert res["worker_off"][-1] > n // 2
    seqs = worker_sequences(res, CONTIG, rng, p_bad=0.05)
    check_join(emu, rows, res, seqs, CONTIG, rng, F.JOIN_CLOSE_PARALLEL, workload + " join", cus=cus)


@pytest.mark.parametrize("seed", [True, False], ids=["seed", "noseed"])
def test_emulated_fork_join_lenient(emu, seed):
    rng = np.random.default_rng(11)
    rows = hand_rows(SCATTERED, [7, 8, 9, 1000, 150000]) + lenient_hand_rows(SCATTERED, [7, 8, 1001, 149999])
    rows += [insert_gaps(r, SCATTERED, rng, p=0.6, max_len=4, keep_last=True).tolist()
             for r in synthetic_main_rows("small", 48, SCATTERED, seed=13)]
    res = check_fork(emu, rows, SCATTERED, seed, rng, "lenient", lenient=True)
    seqs = worker_sequences(res, SCATTERED, rng, p_bad=0.1)
    check_join(emu, rows, res, seqs, SCATTERED, rng, F.JOIN_CLOSE_PARALLEL, "lenient join")


def test_emulated_fork_join_many_rows(emu):
    """More rows than one scan tile: the three-pass scans of the counts."""
    rng = np.random.default_rng(12)
    rows = short_rows(CONTIG, 9001, rng)
    res = check_fork(emu, rows, CONTIG, True, rng, "many rows", cus=4)
    seqs = worker_sequences(res, CONTIG, rng, p_bad=0.05)
    check_join(emu, rows, res, seqs, CONTIG, rng, F.JOIN_CLOSE_PARALLEL, "many rows join", cus=4)


def test_emulated_fork_join_edges(emu):
    """No rows; rows with negative starts or lengths; join worker offsets out
    of order."""
    z = np.zeros(0, np.int64)
    g = emu_fork(emu, np.zeros(1, np.int32), z, np.zeros(0, np.int32), CONTIG, True)
    assert list(g["totals"]) == [0, 0, 0] and list(g["worker_off"]) == [0]
    g = emu_join(emu, (np.zeros(1, np.int32), z, np.zeros(0, np.int32)), [0], (np.zeros(1, np.int32), z,
                                                                                 np.zeros(0, np.int32)), CONTIG, 0)
    assert list(g["totals"]) == [0, 0] and list(g["starts"]) == [0]
    rng = np.random.default_rng(6)
    rows = hand_rows(CONTIG, [7, 8])
    tok, st, ln = layout(rows, rng)
    res, _, _, _ = oracle_fork(rows, CONTIG, True)
    ln2, st2 = ln.copy(), st.copy()
    ln2[0], st2[1] = -5, -1
    g = emu_fork(emu, tok, st2, ln2, CONTIG, True)
    assert g["row_status"][0] == PX.PACK_BAD_ROW and g["row_status"][1] == PX.PACK_BAD_ROW
    assert np.array_equal(g["row_status"][2:], np.array(res["status"][2:], np.uint32))
    seqs = worker_sequences(res, CONTIG, rng)
    off_bad = np.array(res["worker_off"], np.int64)
    off_bad[1] = off_bad[2] + 1
    g = emu_join(emu, (tok, st, ln), off_bad, layout(seqs, rng), CONTIG, F.JOIN_CLOSE_PARALLEL)
    assert g["row_status"][1] & PX.PACK_BAD_ROW and g["lengths"][1] == 0


# ---------------------------------------------------------------- planted mistakes

MUTANTS = {
    # the seed of each entry starts one token late (fork_copy, closed form)
    "seed-offset": ("fork_kernels.h", "ft = o + 2 + 2 * e + (cs - to - e * (L + 1));",
                    "ft = o + 3 + 2 * e + (cs - to - e * (L + 1));"),
    # the carry of earlier scan tiles is dropped (pack_rows)
    "tile-carry": ("fork_kernels.h", "off[k] += a.tile_off[blockIdx.x * K + k];", "off[k] += 0;"),
    # a worker's span starts one token late in the joined row (join_copy)
    "join-span": ("fork_kernels.h", "a.wtokens + __shfl(ws, k, WAVE) + L, s0,", "a.wtokens + __shfl(ws, k, WAVE) + L + 1, s0,"),
}


@pytest.fixture(scope="module")
def mutant_bins(tmp_path_factory):
    base = tmp_path_factory.mktemp("simt_fork_mutants")
    procs, bins = [], {}
    for name, (fname, old, new) in MUTANTS.items():
        d = base / name
        shutil.copytree(CSRC, d)
        p = d / fname
        s = p.read_text()
        assert s.count(old) == 1, name
        p.write_text(s.replace(old, new))
        out = str(base / ("emu_" + name))
        cmd = [CLANG, "-std=c++17", "-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
               "-ffp-contract=off", "-I", SIMT, "-I", os.path.join(ROOT, "include"), "-I", str(d), "-x", "c++",
               str(d / "parason.hip"), str(d / "fork.hip"), os.path.join(SIMT, "emu_fork.cpp"), "-o", out]
        procs.append(subprocess.Popen(cmd))
        bins[name] = out
    assert all(p.wait() == 0 for p in procs)
    return bins


@pytest.mark.parametrize("name", sorted(MUTANTS))
def test_emulated_fork_mutants_caught(mutant_bins, name):
    rng = np.random.default_rng(2)
    caught = False
    try:
        if name == "tile-carry":
            rows = short_rows(CONTIG, 4200, rng)
            check_fork(mutant_bins[name], rows, CONTIG, True, rng, name, cus=4)
        else:
            rows = synthetic_main_rows("small", 32, CONTIG, seed=3)
            res = check_fork(mutant_bins[name], rows, CONTIG, True, rng, name)
            seqs = worker_sequences(res, CONTIG, rng)
            check_join(mutant_bins[name], rows, res, seqs, CONTIG, rng, F.JOIN_CLOSE_PARALLEL, name)
    except (AssertionError, RuntimeError):
        caught = True
    assert caught, name
