"""GPU parity of fork/join packing against the CPU oracle.

Main rows are synthetic rollouts cut right after one of their </Outlines>
tags (so the outlines sit at every depth of nesting and after long text),
plus hand-made rows that the fork must reject, long outlines that span many
256-token chunks, and rows of length 0 and 1.  Every fork output (row status,
worker offsets, each worker's row, entry, kind, context start, length and
tokens) must equal the oracle's exactly; joins of worker sequences laid out
out of order with gaps (some of them malformed on purpose) must equal the
oracle's joined rows exactly, with and without </Parallel> and append-only."""
import numpy as np
import pytest

from fork_cases import (CONTIG, SCATTERED, hand_rows, layout, lenient_hand_rows, oracle_fork, short_rows,
                        synthetic_main_rows, worker_sequences)
from gpu_util import insert_gaps, log, to_dev
from oracle import fork_oracle as F
from paper_2608_24658_amd import parason as PX
from tests import grammar_pins as GP

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu



@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch.device("cuda:0")


def check_fork(dev, px, rows, tags, seed, rng, what, lenient=False):
    tok, st, ln = layout(rows, rng)
    res, exp_starts, exp_lens, exp_flat = oracle_fork(rows, tags, seed, lenient)
    got = px.fork(to_dev(tok, torch.int32, dev), to_dev(st, torch.int64, dev), to_dev(ln, torch.int32, dev), seed=seed)
    torch.cuda.synchronize()
    g = {k: v.cpu().numpy() for k, v in got.items()}
    assert np.array_equal(g["row_status"].view(np.uint32), np.array(res["status"], np.uint32)), what
    assert np.array_equal(g["worker_off"], np.array(res["worker_off"], np.int64)), what
    W = res["worker_off"][-1]
    assert list(g["totals"]) == [W, int(exp_lens.sum()), 0], what
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
    return res, got


def check_join(dev, px, rows, res, seqs, tags, rng, flags, what):
    tok, st, ln = layout(rows, rng)
    wtok, wst, wln = layout(seqs, rng)
    exp, exp_st = F.join(rows, res["worker_off"], seqs, tags, flags=flags)
    got = px.join(to_dev(tok, torch.int32, dev), to_dev(st, torch.int64, dev), to_dev(ln, torch.int32, dev),
                  to_dev(np.array(res["worker_off"], np.int64), torch.int64, dev), to_dev(wtok, torch.int32, dev),
                  to_dev(wst, torch.int64, dev), to_dev(wln, torch.int32, dev),
                  close=bool(flags & F.JOIN_CLOSE_PARALLEL), append_only=bool(flags & F.JOIN_APPEND_ONLY))
    torch.cuda.synchronize()
    g = {k: v.cpu().numpy() for k, v in got.items()}
    assert np.array_equal(g["row_status"].view(np.uint32), np.array(exp_st, np.uint32)), what
    lens = np.array([len(r) for r in exp], np.int64)
    assert np.array_equal(g["lengths"], lens.astype(np.int32)), what
    assert g["starts"][0] == 0 and np.array_equal(np.diff(g["starts"]), lens), what
    flat = np.array([x for r in exp for x in r], np.int32)
    assert np.array_equal(g["tokens"], flat), what
    assert list(g["totals"]) == [int(lens.sum()), 0], what


@pytest.mark.parametrize("tags", [CONTIG, SCATTERED], ids=["contiguous", "scattered"])
@pytest.mark.parametrize("seed", [True, False], ids=["seed", "noseed"])
def test_fork_join_hand_rows(dev, tags, seed):
    log("case fork hand rows tags=%s seed=%s" % (tags[0], seed))
    rng = np.random.default_rng(1)
    px = PX.Parason(tags)
    rows = hand_rows(tags, [7, 8, 9, 1000, 150000])
    res, _ = check_fork(dev, px, rows, tags, seed, rng, "hand")
    assert sum(s == 0 for s in res["status"]) >= 12
    seqs = worker_sequences(res, tags, rng, p_bad=0.2)
    for flags in (F.JOIN_CLOSE_PARALLEL, 0, F.JOIN_APPEND_ONLY, F.JOIN_CLOSE_PARALLEL | F.JOIN_APPEND_ONLY):
        check_join(dev, px, rows, res, seqs, tags, rng, flags, "hand join %d" % flags)


@pytest.mark.parametrize("workload,n", [("small", 256), ("ragged", 512)])
def test_fork_join_synthetic(dev, workload, n):
    log("case fork synthetic %s n=%d" % (workload, n))
    rng = np.random.default_rng(2)
    px = PX.Parason(CONTIG)
    rows = synthetic_main_rows(workload, n, CONTIG, seed=3)
    res, _ = check_fork(dev, px, rows, CONTIG, True, rng, workload)
    assert res["worker_off"][-1] > n // 2
    seqs = worker_sequences(res, CONTIG, rng, p_bad=0.05)
    check_join(dev, px, rows, res, seqs, CONTIG, rng, F.JOIN_CLOSE_PARALLEL, workload + " join")


def test_fork_join_scattered_synthetic(dev):
    log("case fork synthetic scattered")
    rng = np.random.default_rng(4)
    px = PX.Parason(SCATTERED)
    rows = synthetic_main_rows("small", 128, SCATTERED, seed=5)
    res, _ = check_fork(dev, px, rows, SCATTERED, False, rng, "scattered")
    seqs = worker_sequences(res, SCATTERED, rng)
    check_join(dev, px, rows, res, seqs, SCATTERED, rng, F.JOIN_CLOSE_PARALLEL | F.JOIN_APPEND_ONLY, "sc join")


@pytest.mark.parametrize("seed", [True, False], ids=["seed", "noseed"])
def test_fork_join_many_rows(dev, seed):
    """More rows than one scan tile (4096): the scans of the worker and token
    counts take three passes instead of one block."""
    log("case fork many rows seed=%s" % seed)
    rng = np.random.default_rng(12)
    px = PX.Parason(CONTIG)
    rows = short_rows(CONTIG, 9001, rng)
    res, _ = check_fork(dev, px, rows, CONTIG, seed, rng, "many rows")
    assert res["worker_off"][-1] > 9001
    seqs = worker_sequences(res, CONTIG, rng, p_bad=0.05)
    check_join(dev, px, rows, res, seqs, CONTIG, rng, F.JOIN_CLOSE_PARALLEL, "many rows join")


def test_fork_join_no_rows(dev):
    log("case fork/join of zero rows")
    px = PX.Parason(CONTIG)
    z32, z64 = torch.zeros(0, dtype=torch.int32, device=dev), torch.zeros(0, dtype=torch.int64, device=dev)
    got = px.fork(torch.zeros(1, dtype=torch.int32, device=dev), z64, z32, seed=True)
    torch.cuda.synchronize()
    assert list(got["totals"].cpu().numpy()) == [0, 0, 0]
    assert got["worker_off"].cpu().numpy().tolist() == [0]
    got = px.join(torch.zeros(1, dtype=torch.int32, device=dev), z64, z32, torch.zeros(1, dtype=torch.int64, device=dev),
                  torch.zeros(1, dtype=torch.int32, device=dev), z64, z32)
    torch.cuda.synchronize()
    assert list(got["totals"].cpu().numpy()) == [0, 0]
    assert got["starts"].cpu().numpy().tolist() == [0]


def test_fork_capacity_and_bad_rows(dev):
    log("case fork capacity / bad rows")
    px = PX.Parason(CONTIG)
    rows = hand_rows(CONTIG, [7, 8])
    rng = np.random.default_rng(6)
    tok, st, ln = layout(rows, rng)
    res, _, exp_lens, _ = oracle_fork(rows, CONTIG, True)
    W, T = res["worker_off"][-1], int(exp_lens.sum())
    args = (to_dev(tok, torch.int32, dev), to_dev(st, torch.int64, dev), to_dev(ln, torch.int32, dev))
    for mw, cap in ((W - 1, T), (W, T - 1), (0, 0)):
        got = px.fork(*args, seed=True, max_workers=mw, ctx_capacity=cap)
        torch.cuda.synchronize()
        assert list(got["totals"].cpu().numpy()) == [W, T, 1]
        assert np.array_equal(got["worker_off"].cpu().numpy(), np.array(res["worker_off"]))
        assert np.array_equal(got["row_status"].cpu().numpy().view(np.uint32), np.array(res["status"], np.uint32))
    # negative lengths and starts are flagged, never read
    ln2, st2 = ln.copy(), st.copy()
    ln2[0], st2[1] = -5, -1
    got = px.fork(args[0], to_dev(st2, torch.int64, dev), to_dev(ln2, torch.int32, dev), seed=True)
    torch.cuda.synchronize()
    stat = got["row_status"].cpu().numpy().view(np.uint32)
    assert stat[0] == PX.PACK_BAD_ROW and stat[1] == PX.PACK_BAD_ROW
    assert np.array_equal(stat[2:], np.array(res["status"][2:], np.uint32))
    # join: worker offsets out of order or beyond the worker count
    seqs = worker_sequences(res, CONTIG, rng)
    wtok, wst, wln = layout(seqs, rng)
    off = np.array(res["worker_off"], np.int64)
    off_bad = off.copy()
    off_bad[1] = off_bad[2] + 1  # row 0 ends after row 1 begins: row 1 has w1 < w0
    got = px.join(*args, to_dev(off_bad, torch.int64, dev), to_dev(wtok, torch.int32, dev),
                  to_dev(wst, torch.int64, dev), to_dev(wln, torch.int32, dev), capacity=None)
    torch.cuda.synchronize()
    stat = got["row_status"].cpu().numpy().view(np.uint32)
    assert stat[1] & PX.PACK_BAD_ROW and got["lengths"].cpu().numpy()[1] == 0


def test_fork_join_typical_batch(dev):
    """The bench's batch: 1024 rollouts of the typical workload cut at an
    outline.  Every row's outline is parsed by the oracle; every context, worker
    record and joined row is compared.  The worker sequences handed to the join
    are built on the host from the oracle's contexts."""
    log("case fork typical 1024")
    rng = np.random.default_rng(7)
    px = PX.Parason(CONTIG)
    rows = [np.asarray(r, np.int32) for r in synthetic_main_rows("typical", 1024, CONTIG, seed=8, p_raw=0.0)]
    thr, end_thr, end_par = CONTIG[GP.THR - 1], CONTIG[GP.END_THR - 1], CONTIG[GP.END_PAR - 1]
    # oracle: the outline of every row, its contexts (row + <Thread> + entry text)
    status, off, ctx, kinds, w_row, w_entry = [], [0], [], [], [], []
    for i, r in enumerate(rows):
        st, entries = F.parse_outline(r.tolist(), CONTIG)
        status.append(st)
        for k, (kind, a, b) in enumerate(entries):
            ctx.append(np.concatenate([r, np.array([thr], np.int32), r[a:b]]))
            kinds.append(1 if kind == F.SUB else 2)
            w_row.append(i)
            w_entry.append(k)
        off.append(off[-1] + len(entries))
    W = off[-1]
    tok, st, ln = layout(rows, rng)
    got = px.fork(to_dev(tok, torch.int32, dev), to_dev(st, torch.int64, dev), to_dev(ln, torch.int32, dev),
                  seed=True)
    torch.cuda.synchronize()
    g = {k: v.cpu().numpy() for k, v in got.items()}
    assert np.array_equal(g["row_status"].view(np.uint32), np.array(status, np.uint32))
    assert np.array_equal(g["worker_off"], np.array(off, np.int64)) and W > 1024
    assert np.array_equal(g["ctx_row"], np.array(w_row, np.int32))
    assert np.array_equal(g["ctx_entry"], np.array(w_entry, np.int32))
    assert np.array_equal(g["ctx_kind"], np.array(kinds, np.int32))
    lens = np.array([c.size for c in ctx], np.int64)
    starts = np.concatenate([[0], np.cumsum(lens)[:-1]])
    assert np.array_equal(g["ctx_lengths"], lens.astype(np.int32)) and np.array_equal(g["ctx_starts"], starts)
    assert list(g["totals"]) == [W, int(lens.sum()), 0]
    assert np.array_equal(g["ctx_tokens"], np.concatenate(ctx))
    # workers: the oracle's context + generated text + </Thread>, laid out out of order
    seqs = [np.concatenate([c, rng.integers(0, 1000, size=int(rng.integers(0, 60))).astype(np.int32),
                            np.array([end_thr], np.int32)]) for c in ctx]
    wtok, wst, wln = layout(seqs, rng)
    j = px.join(to_dev(tok, torch.int32, dev), to_dev(st, torch.int64, dev), to_dev(ln, torch.int32, dev),
                to_dev(np.array(off, np.int64), torch.int64, dev), to_dev(wtok, torch.int32, dev),
                to_dev(wst, torch.int64, dev), to_dev(wln, torch.int32, dev))
    torch.cuda.synchronize()
    jg = {k: v.cpu().numpy() for k, v in j.items()}
    assert not jg["row_status"].any() and jg["totals"][1] == 0
    exp = [np.concatenate([r] + [seqs[w][r.size:] for w in range(off[i], off[i + 1])] +
                          [np.array([end_par], np.int32)]) for i, r in enumerate(rows)]
    assert np.array_equal(jg["lengths"], np.array([e.size for e in exp], np.int32))
    assert np.array_equal(jg["tokens"], np.concatenate(exp))
    # and the oracle's join itself on a sample of rows
    for i in sorted(rng.choice(1024, size=16, replace=False).tolist()):
        ws = [seqs[w].tolist() for w in range(off[i], off[i + 1])]
        e, est = F.join([rows[i].tolist()], [0, len(ws)], ws, CONTIG)
        assert est == [0] and np.array_equal(np.asarray(e[0], np.int32), exp[i]), i


# --------------------------------------------------------------------------- lenient gaps


@pytest.mark.parametrize("tags", [CONTIG, SCATTERED], ids=["contiguous", "scattered"])
@pytest.mark.parametrize("seed", [True, False], ids=["seed", "noseed"])
def test_fork_join_lenient_hand_rows(dev, tags, seed):
    log("case fork lenient hand rows tags=%s seed=%s" % (tags[0], seed))
    rng = np.random.default_rng(11)
    px = PX.Parason(tags, flags=PX.CFG_LENIENT_GAPS)
    rows = hand_rows(tags, [7, 8, 9, 1000, 150000]) + lenient_hand_rows(tags, [7, 8, 1001, 149999])
    res, _ = check_fork(dev, px, rows, tags, seed, rng, "lenient hand", lenient=True)
    strict = F.fork(rows, tags, flags=F.FORK_SEED_ENTRY if seed else 0)
    assert sum(s == 0 for s in res["status"]) > sum(s == 0 for s in strict["status"]) + 8
    seqs = worker_sequences(res, tags, rng, p_bad=0.1)
    check_join(dev, px, rows, res, seqs, tags, rng, F.JOIN_CLOSE_PARALLEL, "lenient hand join")


@pytest.mark.parametrize("workload,n", [("small", 256), ("ragged", 512)])
def test_fork_join_lenient_synthetic(dev, workload, n):
    log("case fork lenient synthetic %s n=%d" % (workload, n))
    rng = np.random.default_rng(12)
    px = PX.Parason(SCATTERED, flags=PX.CFG_LENIENT_GAPS)
    rows = [insert_gaps(r, SCATTERED, rng, p=0.6, max_len=4, keep_last=True).tolist()
            for r in synthetic_main_rows(workload, n, SCATTERED, seed=13)]
    res, _ = check_fork(dev, px, rows, SCATTERED, True, rng, "lenient " + workload, lenient=True)
    assert res["worker_off"][-1] > n // 2
    seqs = worker_sequences(res, SCATTERED, rng, p_bad=0.05)
    check_join(dev, px, rows, res, seqs, SCATTERED, rng, F.JOIN_CLOSE_PARALLEL, "lenient " + workload + " join")
