"""The accounting kernels run on the CPU, under AddressSanitizer and
UndefinedBehaviorSanitizer, against the oracle.

tests/simt/hip/hip_runtime.h emulates the HIP subset the kernels use (lanes as
fibers meeting at every wave operation: ballot, shuffles, readlane,
readfirstlane, DPP row shifts, ds_bpermute; blocks run one after the other).
The library's own csrc/parason.hip is compiled with it for the host, and the
driver tests/simt/emu_main.cpp runs batches through the C-ABI (parason_run and
parason_run_noalloc) with host memory as device memory.  The emulated device
reports a chosen number of compute units, which picks the kernels a batch
takes: with many units every batch here is small (plan, scan_rows, rows_par,
group_reward); with one or two, rows_fast after gather_rows, then rows_mid and
the single-thread deep tier.  The workspace is handed over filled with a byte
pattern and sized exactly, so reliance on its contents or reads past it fail.

Planted mistakes in copies of the kernel sources (an off-by-one in a DPP
segmented scan, a carry lost inside a lane's events of rows_par's segmented
scan, a lost carry in the scan's compaction, a dropped row-edge mask, an
unreserved pool part, a tag class read from the wrong table nibble, a
dynamic scan chunk that ends a segment early, a block pool chunk that starts
a segment late)
must each be caught by these comparisons."""
import os
import shutil
import subprocess

import numpy as np
import pytest

import grammar_pins as GP
from adversarial import adversarial_streams, deep_stream, fanout_stream, pack
from gpu_util import DEFAULT_COEF, compare, insert_gaps, oracle_expect
from oracle import oracle as O
from paper_2608_24658_amd import parason as PX
from paper_2608_24658_amd.synth import synth as S

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2608_24658_amd", "csrc")
SIMT = os.path.join(ROOT, "tests", "simt")
CLANG = "/opt/rocm/llvm/bin/clang++"
TAGS = S.CONTIGUOUS_TAGS
LOW_IDS = np.array([3, 9, 4, 11, 0, 13, 1, 6, 15, 2, 10, 8], dtype=np.int32)
G = 8
INT_OUT = ("total", "latency", "n_subtask", "n_trial", "n_blocks", "max_depth", "first_error_pos", "flags")
FLOAT_OUT = ("reward", "r_subtask", "r_trial", "eta", "accel")

pytestmark = pytest.mark.skipif(not os.path.exists(CLANG), reason="no host clang++ with the sanitizers")


def build(out, csrc=CSRC):
    cmd = [CLANG, "-std=c++17", "-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
           "-ffp-contract=off", "-I", SIMT, "-I", os.path.join(ROOT, "include"), "-I", csrc, "-x", "c++",
           os.path.join(csrc, "parason.hip"), os.path.join(SIMT, "emu_main.cpp"), "-o", out]
    subprocess.check_call(cmd)
    return out


@pytest.fixture(scope="module")
def emu(tmp_path_factory):
    return build(str(tmp_path_factory.mktemp("simt") / "emu"))


def run_emu(binary, tokens, starts, lengths, correct, tags=TAGS, flags=0, cus=2, shift=0, noalloc=False,
            ws_tokens=None, coef=DEFAULT_COEF, tmp="/tmp"):
    n = len(starts)
    tokens = np.ascontiguousarray(tokens, np.int32)
    if ws_tokens is None:
        ws_tokens = int(np.maximum(np.asarray(lengths), 0).astype(np.int64).sum())
    hdr = (np.array([n, tokens.size, ws_tokens], np.int64).tobytes() + np.asarray(tags, np.int32).tobytes()
           + np.array([G], np.int32).tobytes() + np.array([flags], np.uint32).tobytes()
           + np.array([cus, shift, int(noalloc)], np.int32).tobytes()
           + np.array([coef[k] for k in ("alpha", "beta_subtask", "beta_trial", "rho", "rho_clip")],
                      np.float64).tobytes())
    body = (tokens.tobytes() + np.asarray(starts, np.int64).tobytes() + np.asarray(lengths, np.int32).tobytes()
            + np.asarray(correct, np.uint8).tobytes())
    fin = os.path.join(tmp, "emu_in_%d.bin" % os.getpid())
    fout = os.path.join(tmp, "emu_out_%d.bin" % os.getpid())
    with open(fin, "wb") as f:
        f.write(hdr + body)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:halt_on_error=1:abort_on_error=1",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    r = subprocess.run([binary, fin, fout], env=env, capture_output=True, text=True, timeout=600)
    if r.returncode != 0:
        raise RuntimeError("emulation failed (%d):\n%s" % (r.returncode, r.stderr[-4000:]))
    b = open(fout, "rb").read()
    os.unlink(fin)
    os.unlink(fout)
    out, off = {}, 0
    for k in INT_OUT:
        out[k] = np.frombuffer(b, np.int32, n, off).copy()
        off += 4 * n
    out["flags"] = out["flags"].view(np.uint32)
    for k in FLOAT_OUT:
        out[k] = np.frombuffer(b, np.float32, n, off).copy()
        off += 4 * n
    out["saved"] = np.frombuffer(b, np.int32, n, off).copy()
    off += 4 * n
    return out, int(np.frombuffer(b, np.int32, 1, off)[0])


def check(binary, tokens, starts, lengths, correct, tags=TAGS, flags=0, cus=2, what="", **kw):
    got, rc = run_emu(binary, tokens, starts, lengths, correct, tags, flags, cus, **kw)
    assert rc == PX.OK, (what, rc)
    exp = oracle_expect(tokens, starts, lengths, correct, tags, G, DEFAULT_COEF, flags & ~PX.CFG_TAG_COMPARE)
    compare(got, *exp, what=what, exact_reward=not (flags & PX.CFG_BATCH_STATS))
    return got


# rows_par for every batch here (fewer rows than 20 waves per emulated unit x 2)
MANY = 64
# rows_fast (one row per lane), gather_rows, rows_mid, deep tier
FEW = 1


@pytest.mark.parametrize("workload", ["tiny", "small", "ragged"])
@pytest.mark.parametrize("cus", [MANY, FEW])
def test_emulated_workloads(emu, workload, cus):
    P = S.make_params(workload)
    n = S.n_rows_of(workload)
    tok, st, ln, co = S.host_batch(P, n)
    check(emu, tok, st, ln, co, cus=cus, what="%s cus %d" % (workload, cus))


@pytest.mark.parametrize("n", [2048, 2056])
def test_emulated_plan_boundary(emu, n):
    """With 64 emulated units a batch of 2,048 rows takes rows_par with the
    plan made by the scan blocks, one of 2,056 rows takes rows_par after the
    plan launch (short rows, so the batch stays small)."""
    streams = adversarial_streams()
    streams = [streams[i % len(streams)] for i in range(n)]
    tokens, starts, lengths = pack(streams, TAGS)
    correct = (np.arange(n) % 3 != 0).astype(np.uint8)
    check(emu, tokens, starts, lengths, correct, cus=MANY, what="plan boundary %d" % n)


def stretch(stream, total, rng):
    """The stream with Text runs inserted after tags that Text may follow
    (<think>, </Parallel>, <Thread>, entry openings), about `total` tokens in
    all, so that its events spread over hundreds of segments."""
    spots = [i for i, c in enumerate(stream) if c in (GP.THINK, GP.END_PAR, GP.THR, GP.SUB, GP.TRI)]
    runs = rng.multinomial(total, np.ones(len(spots)) / len(spots))
    out, last = [], 0
    for i, r in zip(spots, runs):
        out += stream[last: i + 1] + [GP.TEXT] * int(r)
        last = i + 1
    return out + stream[last:]


@pytest.mark.parametrize("n,cus", [(8, MANY), (2056, MANY), (64, FEW)])
def test_emulated_rows_without_tokens(emu, n, cus):
    """Batches of empty rows only (not one token): the scan has no segment to
    read, and each batch path (the scan's own plan, the plan launch with
    rows_par, the per-lane row tiers) still writes every row's outputs."""
    tokens = np.zeros(0, np.int32)
    starts = np.zeros(n, np.int64)
    lengths = np.zeros(n, np.int32)
    correct = (np.arange(n) % 2).astype(np.uint8)
    got = check(emu, tokens, starts, lengths, correct, cus=cus, what="empty rows n %d cus %d" % (n, cus))
    assert np.all(got["total"] == 0)


def test_emulated_long_split_rows(emu):
    """Rows of 270k-600k tokens whose events spread over more than 256 (and 512)
    segments, so that rows_par gathers a split row in several chunks of
    segments, some rows with more than 256 events (two event passes)."""
    rng = np.random.default_rng(3)
    streams = [stretch(fanout_stream(40), 300000, rng), stretch(deep_stream(4), 280000, rng),
               stretch(fanout_stream(70), 600000, rng), stretch(fanout_stream(100, 90), 270000, rng),
               stretch(deep_stream(12, GP.TRI), 330000, rng), stretch(fanout_stream(3), 520000, rng)]
    tokens, starts, lengths = pack(streams, TAGS)
    correct = (np.arange(lengths.size) % 2 == 0).astype(np.uint8)
    check(emu, tokens, starts, lengths, correct, cus=MANY, what="long split rows")


def dynamic_batch():
    """2,000 rows of 2,000-5,000 tokens (6.9e6 tokens): on one emulated unit
    (16 scan waves) more than 256 segments per wave, so the scan takes 13/16
    of an equal share per wave, then chunks of the rest in segment order: one
    round of one chunk per wave (c0 = (S - S1) / 32 of about 50 segments), then
    32-segment chunks.  Rows cut by chunk boundaries take the split-row path."""
    P = S.make_params("small")
    tok, st, ln, co = S.host_batch(P, 2000)
    segs = int(np.sum((ln.astype(np.int64) + 1023) // 1024))  # a lower bound of the scan's segments
    s_dyn = segs * 3 // 16
    assert segs >= 256 * 16 and s_dyn // 32 >= 32, "the batch must reach the dynamic rounds"
    return tok, st, ln, co


def test_emulated_dynamic_scan(emu):
    tok, st, ln, co = dynamic_batch()
    check(emu, tok, st, ln, co, cus=FEW, what="dynamic scan")


BLOCK_POOL_CUS = 16


def block_pool_batch(n=632, cus=BLOCK_POOL_CUS):
    """n rows of 2,000-5,000 tokens on `cus` emulated units take the scan that
    plans the batch itself (2 cus blocks of 8 waves, rows_par after it) with
    more than 64 segments per block, so each block's waves scan equal shares
    of 13/16 of its segments and take the rest two at a time from the block's
    LDS counter."""
    assert n / 2 < cus * 20 and n <= 2048, "the batch must take rows_par and the planning scan"
    P = S.make_params("small")
    tok, st, ln, co = S.host_batch(P, n)
    segs = int(np.sum((ln.astype(np.int64) + 1023) // 1024))  # a lower bound of the scan's segments
    assert segs >= 64 * 2 * cus, "every block must reach its pool"
    return tok, st, ln, co


@pytest.mark.parametrize("n,cus", [(632, 16), (472, 12)])  # 32 blocks (shifts), 24 blocks (divisions)
def test_emulated_block_pool(emu, n, cus):
    tok, st, ln, co = block_pool_batch(n, cus)
    check(emu, tok, st, ln, co, cus=cus, what="block pool %d rows, %d units" % (n, cus))


@pytest.mark.parametrize("tags", ["contiguous", "scattered", "scattered-compare", "low-ids"])
@pytest.mark.parametrize("cus", [16, FEW])
def test_emulated_adversarial(emu, tags, cus):
    """Every short valid string and mutations, nesting to depth 1000, outlines
    beyond 64 entries, all-tag rows whose segments overflow their event
    storage (the dense path, classified again token by token)."""
    tag_ids = {"contiguous": TAGS, "low-ids": LOW_IDS}.get(tags, S.SCATTERED_TAGS)
    tokens, starts, lengths = pack(adversarial_streams(), tag_ids)
    n = lengths.size
    correct = (np.arange(n) % 3 != 0).astype(np.uint8)
    flags = PX.CFG_TAG_COMPARE if tags == "scattered-compare" else 0
    got = check(emu, tokens, starts, lengths, correct, tag_ids, flags, cus, what="adversarial %s" % tags)
    assert int(np.sum(got["max_depth"] == 1000)) == 1


def test_emulated_lenient_gaps(emu):
    rng = np.random.default_rng(21)
    P = S.make_params("small")
    tok, st, ln, co = S.host_batch(P, 64)
    rows = [insert_gaps(tok[st[i]: st[i] + ln[i]], TAGS, rng) for i in range(64)]
    lengths = np.array([r.size for r in rows], np.int32)
    starts = np.zeros(64, np.int64)
    starts[1:] = np.cumsum(lengths[:-1])
    tokens = np.concatenate(rows)
    for cus in (MANY, FEW):
        check(emu, tokens, starts, lengths, co, flags=PX.CFG_LENIENT_GAPS, cus=cus, what="lenient cus %d" % cus)


def test_emulated_layouts_noalloc_batch_stats(emu):
    P = S.make_params("small")
    tok, st, ln, co = S.host_batch(P, 64)
    for shift in (1, 2, 3):
        check(emu, tok, st, ln, co, cus=MANY, shift=shift, what="shift %d" % shift)
    lmax = int(ln.max()) + 3
    padded = np.full((64, lmax), 11, np.int32)
    for i in range(64):
        padded[i, : ln[i]] = tok[st[i]: st[i] + ln[i]]
    check(emu, padded.ravel(), (np.arange(64) * lmax).astype(np.int64), ln, co, cus=FEW, what="padded")
    check(emu, tok, st, ln, co, cus=MANY, noalloc=True, what="noalloc")
    check(emu, tok, st, ln, co, flags=PX.CFG_BATCH_STATS, cus=FEW, what="batch stats")


def test_emulated_bad_rows_and_workspace_overflow(emu):
    P = S.make_params("typical")
    tok, st, ln, co = S.host_batch(P, 16)
    got, rc = run_emu(emu, tok, st, ln, co, cus=MANY, ws_tokens=0)
    assert rc == PX.OK and np.all(got["flags"] == PX.FLAG_WS_OVERFLOW) and np.all(np.isnan(got["reward"]))
    bad = ln.copy()
    bad[3] = -4
    got, rc = run_emu(emu, tok, st, bad, co, cus=MANY)
    assert rc == PX.OK and got["flags"][3] == PX.FLAG_BAD_ROW and np.all(np.isnan(got["reward"][:8]))
    keep = np.r_[8:16]
    exp = oracle_expect(tok, st[keep], ln[keep], co[keep], TAGS, G, DEFAULT_COEF)
    compare({k: v[keep] for k, v in got.items()}, *exp, what="bad-row rest")


MUTANTS = {
    # a dynamic chunk of the scan that ends one segment early (that segment is never scanned)
    "dyn-chunk-gap": ("parason_kernels.h", "e = b + (c0 >> r);", "e = b + (c0 >> r) - 1;"),
    # a block's pool chunks that start one segment late (a segment of a small batch is never scanned)
    "block-chunk-skip": ("parason_kernels.h", "b = uniform64(Bk + L1 + (int64_t)j * BLK_CHUNK);",
                         "b = uniform64(Bk + L1 + 1 + (int64_t)j * BLK_CHUNK);"),
    # a DPP segmented scan whose carry out of the first row of 16 lanes is read one lane early
    "seg-scan-off-by-one": ("device_common.h",
                            "const int32_t v0 = __builtin_amdgcn_readlane(v, 15), v1",
                            "const int32_t v0 = __builtin_amdgcn_readlane(v, 14), v1"),
    # the scan's compaction forgets the count of tags of the vector's first token column
    "compaction-carry": ("parason_kernels.h",
                         "cnt += (uint32_t)(__popcll(b[0]) + __popcll(b[1])",
                         "cnt += (uint32_t)(0 + __popcll(b[1])"),
    # the per-lane form of the segmented scan drops the carry into a lane's
    # second to fourth events (rows_par, four events per lane)
    "lane-carry": ("parason_kernels.h", "if (!seen) v[k] = Op::f(in, v[k]);",
                   "if (!seen && k == 0) v[k] = Op::f(in, v[k]);"),
    # a row's edge segments keep tags of the neighbouring rows
    "edge-mask": ("parason_kernels.h",
                  "if (EDGE) hit = hit && q0 + j >= q_lo && q0 + j < q_hi;",
                  "if (EDGE) hit = hit && q0 + j < q_hi;"),
    # a compact list's pool part is not reserved, so the next list overwrites it
    "pool-cursor": ("parason_kernels.h", "    rc.pc += need;\n}", "    rc.pc += 0 * need;\n}"),
    # the class of a stored tag read from the neighbouring nibble of the table
    "tag-class": ("parason_kernels.h", "(lut >> (4u * ((uint32_t)t - (uint32_t)tm.base)))",
                  "(lut >> (4u * ((uint32_t)t - (uint32_t)tm.base + 1u)))"),
}


def test_planted_mistakes_are_caught(tmp_path):
    """Each mutant (built in parallel) must fail at least one comparison."""
    procs = {}
    for name, (f, old, new) in sorted(MUTANTS.items()):
        d = tmp_path / name
        shutil.copytree(CSRC, d)
        src = (d / f).read_text()
        assert src.count(old) == 1, "the planted line of %s is not in %s" % (name, f)
        (d / f).write_text(src.replace(old, new))
        out = str(tmp_path / (name + ".emu"))
        cmd = [CLANG, "-std=c++17", "-O1", "-g", "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
               "-ffp-contract=off", "-I", SIMT, "-I", os.path.join(ROOT, "include"), "-I", str(d), "-x", "c++",
               str(d / "parason.hip"), os.path.join(SIMT, "emu_main.cpp"), "-o", out]
        procs[name] = (subprocess.Popen(cmd), out)
    for name, (p, _) in procs.items():
        assert p.wait() == 0, name
    P = S.make_params("small")
    tok, st, ln, co = S.host_batch(P, 64)
    tokens, starts, lengths = pack(adversarial_streams(), TAGS)
    correct = (np.arange(lengths.size) % 3 != 0).astype(np.uint8)
    dyn = dynamic_batch()
    blk = block_pool_batch()
    for name, (_, binary) in sorted(procs.items()):
        caught = 0
        configs = [((tok, st, ln, co), MANY), ((tokens, starts, lengths, correct), 16), ((tok, st, ln, co), FEW)]
        if name.startswith("dyn-"):
            configs = [(dyn, FEW)]  # only a large batch takes the dynamic chunks
        if name.startswith("block-"):
            configs = [(blk, BLOCK_POOL_CUS)]  # a planned batch with blocks of at least 64 segments
        for args, cus in configs:
            try:
                check(binary, *args, cus=cus, what=name)
            except (AssertionError, RuntimeError):
                caught += 1
        assert caught > 0, "planted mistake %s went unnoticed" % name
