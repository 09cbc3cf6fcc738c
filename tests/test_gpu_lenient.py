"""GPU parity of the accounting path with lenient gaps (PARASON_CFG_LENIENT_GAPS).

Rows of the seeded workloads get runs of Text after the tags that open a gap
in a parallel region (the line breaks of Figure 3); the HIP path in lenient
mode must match the oracle in lenient mode, and in strict mode the oracle in
strict mode (an error at the first gap).  Hand-built rows cover gaps across
segment boundaries, gaps in deeply nested rows (all three tiers of the row
kernel) and in rows with more than 64 outline entries.  Integer outputs
bit-exact, floats within the bound stated in gpu_util.
"""
import json
import os

import numpy as np
import pytest

import grammar_pins as GP
from gpu_util import DEFAULT_COEF, compare, insert_gaps, log, oracle_expect, run_gpu, to_dev
from oracle import oracle as O
from paper_2608_24658_amd import parason as PX
from paper_2608_24658_amd.synth import synth as S

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

G = S.GROUP_SIZE
LENIENT = PX.CFG_LENIENT_GAPS
assert LENIENT == O.CFG_LENIENT_GAPS


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch.device("cuda:0")


def packed(rows):
    lengths = np.array([len(r) for r in rows], np.int32)
    starts = np.zeros(len(rows), np.int64)
    starts[1:] = np.cumsum(lengths[:-1].astype(np.int64))
    tokens = np.concatenate([np.asarray(r, np.int32) for r in rows]) if lengths.sum() else np.zeros(1, np.int32)
    return tokens, starts, lengths


def run_both(dev, tokens, starts, lengths, correct, tags, what, coef=DEFAULT_COEF):
    """Lenient and strict handles on the same rows, each against the oracle in
    the same mode.  Returns the lenient outputs."""
    args = (to_dev(tokens, torch.int32, dev), to_dev(starts, torch.int64, dev), to_dev(lengths, torch.int32, dev),
            to_dev(correct, torch.uint8, dev))
    out = {}
    for fl in (LENIENT, 0):
        px = PX.Parason(tags, group_size=G, flags=fl, **coef)
        got = run_gpu(px, *args)
        compare(got, *oracle_expect(tokens, starts, lengths, correct, tags, G, coef, fl),
                what="%s %s" % (what, "lenient" if fl else "strict"))
        out[fl] = got
    return out[LENIENT], out[0]


@pytest.mark.parametrize("workload,tags", [("small", "contiguous"), ("ragged", "scattered"),
                                           ("typical", "contiguous")])
def test_workload_with_gaps(dev, workload, tags):
    log("case lenient workload=%s tags=%s" % (workload, tags))
    tag_ids = S.CONTIGUOUS_TAGS if tags == "contiguous" else S.SCATTERED_TAGS
    P = S.make_params(workload, tag_ids=tag_ids)
    n = S.n_rows_of(workload)
    tok, st, ln, co = S.host_batch(P, n)
    rng = np.random.default_rng(21)
    rows = [insert_gaps(tok[st[i]: st[i] + ln[i]], tag_ids, rng, p=0.5, max_len=3) for i in range(n)]
    tokens, starts, lengths = packed(rows)
    got, strict = run_both(dev, tokens, starts, lengths, co, tag_ids, workload)
    valid = (got["flags"] & PX.FLAG_VALID) != 0
    gapped = lengths != ln
    # the gaps are accepted in lenient mode, and every row with one is rejected in strict mode
    assert int(np.sum(valid & gapped)) > n // 3
    assert not np.any(strict["flags"][gapped] & PX.FLAG_VALID)
    log("%s: %d rows, %d with gaps, %d valid in lenient mode" % (workload, n, int(gapped.sum()),
                                                                   int(valid.sum())))


def deep_stream(depth, gap):
    s = [GP.THINK]
    for _ in range(depth):
        s += [GP.PAR] + [GP.TEXT] * gap + [GP.OUT, GP.SUB, GP.TEXT, GP.END_SUB] + [GP.TEXT] * gap + [
            GP.END_OUT] + [GP.TEXT] * gap + [GP.THR, GP.TEXT]
    for _ in range(depth):
        s += [GP.END_THR] + [GP.TEXT] * gap + [GP.END_PAR]
    return s + [GP.END_THINK]


def fanout_stream(k, gap):
    s = [GP.THINK, GP.TEXT, GP.PAR, GP.OUT] + [GP.TEXT] * gap
    for i in range(k):
        s += ([GP.TRI, GP.TEXT, GP.END_TRI] if i % 3 == 0 else [GP.SUB, GP.TEXT, GP.TEXT, GP.END_SUB]) + \
            [GP.TEXT] * (i % (gap + 1))
    s += [GP.END_OUT] + [GP.TEXT] * gap
    for i in range(k):
        s += [GP.THR] + [GP.TEXT] * (i % 5) + [GP.END_THR] + [GP.TEXT] * (i % 2)
    return s + [GP.END_PAR, GP.END_THINK]


def hand_streams():
    streams = []
    strings = [list(s) for s in GP.enumerate_valid(15, "lenient")]
    streams += strings[::5]
    rng = np.random.default_rng(5)
    for s in strings[::23]:  # truncations and one-token mutations
        i = int(rng.integers(0, len(s)))
        streams.append(s[:i] + [int(rng.integers(0, 13))] + s[i + 1:])
        streams.append(s[: int(rng.integers(0, len(s) + 1))])
    # nesting through the three tiers of the row kernel, with gaps at every level
    streams += [deep_stream(d, g) for d, g in ((3, 1), (5, 2), (6, 1), (20, 3), (33, 1), (34, 2), (60, 1))]
    # more than 64 outline entries (the deep store), gaps between them
    streams += [fanout_stream(64, 2), fanout_stream(90, 3)]
    # gaps long enough to span segments (1024 tokens) and to cross their edges
    long = [GP.THINK] + [GP.TEXT] * 1019 + [GP.PAR] + [GP.TEXT] * 3000 + [GP.OUT, GP.SUB, GP.TEXT, GP.END_SUB] + \
        [GP.TEXT] * 2047 + [GP.END_OUT] + [GP.TEXT] * 5 + [GP.THR] + [GP.TEXT] * 4000 + [GP.END_THR] + \
        [GP.TEXT] * 1024 + [GP.THR, GP.END_THR, GP.END_PAR, GP.END_THINK]
    streams.append(long)
    streams.append(long[:1021] + [GP.THINK] + long[1021:])  # a tag inside a gap
    g = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "fig3_repaired_line_breaks.json")))
    streams.append(GP.parse_names(g["stream"]))
    return streams, g


@pytest.mark.parametrize("tags", ["contiguous", "scattered"])
def test_hand_streams_with_gaps(dev, tags):
    log("case lenient hand streams tags=%s" % tags)
    tag_ids = S.CONTIGUOUS_TAGS if tags == "contiguous" else S.SCATTERED_TAGS
    streams, golden = hand_streams()
    while len(streams) % G:
        streams.append(GP.parse_names("think t2 /think"))
    rng = np.random.default_rng(9)
    rows = []
    for s in streams:
        t = np.array(GP.to_tokens(s, tag_ids, 7), np.int32)
        text = rng.integers(0, 150000, size=t.size).astype(np.int32)
        text = np.where(np.isin(text, tag_ids), 7, text)
        rows.append(np.where(np.array([c == GP.TEXT for c in s], bool), text, t) if len(s) else t)
    tokens, starts, lengths = packed(rows)
    correct = (np.arange(len(rows)) % 4 != 0).astype(np.uint8)
    got, _ = run_both(dev, tokens, starts, lengths, correct, tag_ids, "hand")
    i = len(hand_streams()[0]) - 1  # the golden is the last hand stream (before the padding rows)
    for k, v in golden["expected"].items():
        assert int(got[k][i]) == v, k
    assert int(np.max(got["max_depth"])) == 60


def test_many_rows_with_gaps(dev):
    """24,576 rows (more than the one-wave-per-row kernel takes): the lenient
    form of the per-lane automaton, several rows per wave."""
    log("case lenient many rows")
    tag_ids = S.CONTIGUOUS_TAGS
    P = S.make_params("small", tag_ids=tag_ids)
    n0 = S.n_rows_of("small")
    tok, st, ln, co = S.host_batch(P, n0)
    rng = np.random.default_rng(31)
    rows = []
    for rep in range(96):
        for i in range(n0):
            rows.append(insert_gaps(tok[st[i]: st[i] + ln[i]], tag_ids, rng, p=0.3, max_len=2))
    tokens, starts, lengths = packed(rows)
    correct = np.tile(co, 96)
    got, _ = run_both(dev, tokens, starts, lengths, correct, tag_ids, "many rows")
    assert len(rows) == 24576 and int(np.sum(got["flags"] & PX.FLAG_VALID)) > 20000
