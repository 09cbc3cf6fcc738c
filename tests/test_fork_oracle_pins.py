"""Pins of the fork/join oracle (CPU only).

* worked example: the outline of the 24-puzzle trace (Figure 3, Sec. 3.2),
  three <Subtask> entries, written out by hand;
* round trip: in every valid stream up to 14 tokens (and in random larger
  ones), cutting a <Parallel> block at its </Outlines> and handing each of its
  threads back as a worker's output must rebuild the stream up to the block's
  </Parallel> -- the threads are found by an independent bracket matcher;
* the local outline check agrees with an Earley recognizer on
  "<think> <Parallel> <Outlines> ... </Outlines>" for every class string of the
  outline region up to 5 tokens and on 20,000 random longer regions;
* the joined stream is accepted by the accounting parser with as many threads
  as entries.
"""
import itertools
import random

import pytest

from oracle import fork_oracle as F
from oracle import oracle as O
from tests import grammar_pins as GP

TAGS = list(range(100, 112))
TEXT_ID = 7


def toks(classes, text=TEXT_ID):
    return GP.to_tokens(classes, TAGS, text)


def blocks_of(classes):
    """Every <Parallel> block of a valid class string: (pos of </Outlines>,
    thread spans [(start, end_inclusive)], pos of </Parallel>, entry count)."""
    out, stack = [], []
    for p, c in enumerate(classes):
        if c == GP.PAR:
            stack.append(dict(outl=None, threads=[], open_thr=None, entries=0))
        elif c in (GP.SUB, GP.TRI):
            stack[-1]["entries"] += 1
        elif c == GP.END_OUT:
            stack[-1]["outl"] = p
        elif c == GP.THR:
            stack[-1]["threads"].append([p, None])
        elif c == GP.END_THR:
            # the innermost block with an open thread owns this close
            for b in reversed(stack):
                if b["threads"] and b["threads"][-1][1] is None:
                    b["threads"][-1][1] = p
                    break
        elif c == GP.END_PAR:
            b = stack.pop()
            out.append((b["outl"], [tuple(t) for t in b["threads"]], p, b["entries"]))
    return out


def test_worked_example_24_puzzle():
    row = GP.parse_names("think t5 Par Out Sub t3 /Sub Sub t2 /Sub Sub t4 /Sub /Out")
    ids = list(range(200, 200 + len(row)))  # distinct text ids, so seeds are recognisable
    tok = [TAGS[c - 1] if c else ids[p] for p, c in enumerate(row)]
    res = F.fork([tok], TAGS)
    assert res["status"] == [0] and res["worker_off"] == [0, 3]
    assert res["kind"] == [F.SUB] * 3 and res["entry"] == [0, 1, 2] and res["row"] == [0, 0, 0]
    thr = TAGS[GP.THR - 1]
    assert res["ctx"][0] == tok + [thr] + ids[9:12]
    assert res["ctx"][1] == tok + [thr] + ids[14:16]
    assert res["ctx"][2] == tok + [thr] + ids[18:22]
    plain = F.fork([tok], TAGS, flags=0)
    assert plain["ctx"] == [tok + [thr]] * 3


def _round_trip(classes, text_ids=None):
    tok = toks(classes) if text_ids is None else [TAGS[c - 1] if c else text_ids[p] for p, c in enumerate(classes)]
    n_checked = 0
    for outl, threads, endp, n_entries in blocks_of(classes):
        if len(threads) != n_entries:
            continue  # a runtime dispatches exactly one worker per entry
        main = tok[:outl + 1]
        res = F.fork([main], TAGS, flags=0)
        assert res["status"] == [0] and res["worker_off"] == [0, n_entries]
        seqs = [main + tok[a:b + 1] for a, b in threads]
        for c, s in zip(res["ctx"], seqs):
            assert s[:len(c)] == c  # each worker's sequence extends its context
        joined, st = F.join([main], res["worker_off"], seqs, TAGS)
        assert st == [0]
        assert joined[0] == tok[:endp + 1]
        app, _ = F.join([main], res["worker_off"], seqs, TAGS, flags=F.JOIN_CLOSE_PARALLEL | F.JOIN_APPEND_ONLY)
        assert app[0] == tok[outl + 1:endp + 1]
        n_checked += 1
    return n_checked


def test_round_trip_all_short_streams():
    n = 0
    for s in GP.enumerate_valid(14):
        n += _round_trip(list(s))
    assert n > 20


def test_round_trip_random_nested_streams():
    rng = random.Random(5)
    n = 0
    for _ in range(150):
        cls = [GP.THINK]

        def body(depth):
            out = []
            for _ in range(rng.randrange(0, 3)):
                if depth < 3 and rng.random() < 0.5:
                    k = rng.randrange(1, 4)
                    out += [GP.PAR, GP.OUT]
                    for _ in range(k):
                        e = rng.choice([GP.SUB, GP.TRI])
                        out += [e] + [GP.TEXT] * rng.randrange(1, 4) + [e + 1]
                    out += [GP.END_OUT]
                    for _ in range(k):
                        out += [GP.THR] + body(depth + 1) + [GP.END_THR]
                    out += [GP.END_PAR]
                else:
                    out += [GP.TEXT] * rng.randrange(1, 5)
            return out

        cls += body(0) + [GP.END_THINK]
        assert GP.earley(cls)[0]
        n += _round_trip(cls, text_ids=[rng.randrange(0, 99) for _ in cls])
    assert n > 50


def test_round_trip_with_seeded_threads():
    # threads that begin with their entry's text extend the seeded contexts
    rng = random.Random(9)
    for _ in range(50):
        k = rng.randrange(1, 5)
        main_cls = [GP.THINK, GP.TEXT, GP.PAR, GP.OUT]
        for _ in range(k):
            e = rng.choice([GP.SUB, GP.TRI])
            main_cls += [e] + [GP.TEXT] * rng.randrange(1, 5) + [e + 1]
        main_cls += [GP.END_OUT]
        ids = [rng.randrange(0, 99) for _ in main_cls]
        main = [TAGS[c - 1] if c else ids[p] for p, c in enumerate(main_cls)]
        res = F.fork([main], TAGS)
        assert res["worker_off"] == [0, k]
        seqs = []
        for w in range(k):
            extra = [rng.randrange(0, 99) for _ in range(rng.randrange(0, 4))]
            seqs.append(res["ctx"][w] + extra + [TAGS[GP.END_THR - 1]])
        joined, st = F.join([main], res["worker_off"], seqs, TAGS)
        assert st == [0]
        full = joined[0] + [TAGS[GP.END_THINK - 1]]
        r = O.eval_stream(full, TAGS)
        assert r["flags"] & O.F_VALID and not r["flags"] & O.F_COUNT_MISMATCH
        assert r["n_blocks"] == 1


REGION_CLASSES = [GP.TEXT, GP.SUB, GP.END_SUB, GP.TRI, GP.END_TRI, GP.OUT, GP.PAR, GP.THR]


def _regions():
    for n in range(0, 6):  # every region of up to 5 classes
        for region in itertools.product(REGION_CLASSES, repeat=n):
            yield list(region)
    rng = random.Random(3)
    for _ in range(20000):  # and random longer ones, biased to well-formed entries
        region = []
        while len(region) < 12 and rng.random() < 0.85:
            if rng.random() < 0.8:
                e = rng.choice([GP.SUB, GP.TRI])
                region += [e] + [GP.TEXT] * rng.randrange(0, 3) + [rng.choice([e + 1, e + 1, e + 1, GP.END_SUB])]
            else:
                region.append(rng.choice(REGION_CLASSES))
        yield region


def test_outline_check_matches_earley():
    n_ok = 0
    for region in _regions():
        row = [GP.THINK, GP.PAR, GP.OUT] + region + [GP.END_OUT]
        st, entries = F.parse_outline(toks(row), TAGS)
        # the last <Outlines> of the row opens the dispatched outline
        o = max(p for p, c in enumerate(row[:-1]) if c == GP.OUT)
        local = [GP.THINK] + row[o - 1:]
        ok, pos = GP.earley(local)
        viable = ok or pos == len(local)
        assert (st == 0) == (viable and row[o - 1] == GP.PAR), [GP.NAMES[c] for c in row]
        if st == 0:
            assert len(entries) == sum(1 for c in row[o:] if c in (GP.SUB, GP.TRI))
            n_ok += 1
    assert n_ok > 10


@pytest.mark.parametrize("names,status", [
    ("think Par Out Sub t /Sub", F.ST_NO_OUTLINE_END),
    ("", F.ST_NO_OUTLINE_END),
    ("think t /Out", F.ST_NO_OUTLINE),
    ("think Out Sub t /Sub /Out", F.ST_NO_OUTLINE),
    ("think Par t Out Sub t /Sub /Out", F.ST_NO_OUTLINE),
    ("think Par Out /Out", F.ST_BAD_ENTRY),
    ("think Par Out Sub /Sub /Out", F.ST_BAD_ENTRY),
    ("think Par Out Sub t /Tri /Out", F.ST_BAD_ENTRY),
    ("think Par Out Sub t /Sub t Tri t /Tri /Out", F.ST_BAD_ENTRY),
    ("think Par Out t Sub t /Sub /Out", F.ST_BAD_ENTRY),
    ("think Par Out Sub t Thr /Sub /Out", F.ST_BAD_ENTRY),
])
def test_rejected_rows(names, status):
    res = F.fork([toks(GP.parse_names(names))], TAGS)
    assert res["status"] == [status] and res["worker_off"] == [0, 0] and res["ctx"] == []


def test_join_flags_bad_threads():
    main = toks(GP.parse_names("think Par Out Sub t /Sub Tri t /Tri /Out"))
    thr, ethr = TAGS[GP.THR - 1], TAGS[GP.END_THR - 1]
    good = main + [thr, 7, ethr]
    for bad in (main + [7, ethr], main + [thr, 7], main + [thr], main):
        out, st = F.join([main], [0, 2], [good, bad], TAGS)
        assert st == [F.ST_BAD_THREAD]
        assert out[0] == main + good[len(main):] + bad[len(main):] + [TAGS[GP.END_PAR - 1]]
    out, st = F.join([main], [0, 2], [good, good], TAGS, flags=0)
    assert st == [0] and out[0] == main + [thr, 7, ethr] * 2


# --------------------------------------------------------------------------- lenient gaps
# With the lenient-gaps reading, Text may stand between <Parallel> and
# <Outlines>, after <Outlines>, between entries and before </Outlines> (and
# after </Outlines> and every thread, which the fork never sees).


def test_outline_check_matches_earley_lenient():
    rng = random.Random(11)
    n_ok = n_gap = 0
    for region in _regions():
        pre = [GP.TEXT] * rng.choice([0, 0, 1, 2])
        row = [GP.THINK, GP.PAR] + pre + [GP.OUT] + region + [GP.END_OUT]
        st, entries = F.parse_outline(toks(row), TAGS, lenient=True)
        o = max(p for p, c in enumerate(row[:-1]) if c == GP.OUT)
        q = o - 1
        while q >= 0 and row[q] == GP.TEXT:
            q -= 1
        local = [GP.THINK] + row[q:]
        ok, pos = GP.earley(local, "lenient")
        viable = ok or pos == len(local)
        assert (st == 0) == (viable and row[q] == GP.PAR), [GP.NAMES[c] for c in row]
        if st == 0:
            assert len(entries) == sum(1 for c in row[o:] if c in (GP.SUB, GP.TRI))
            for kind, a, b in entries:  # the seed is exactly the entry's text
                assert row[a - 1] == kind and row[b] == kind + 1 and set(row[a:b]) == {GP.TEXT}
            n_ok += 1
            n_gap += not GP.earley(local)[0] and GP.earley(local)[1] != len(local)
    assert n_ok > 10 and n_gap > 10


def _round_trip_lenient(classes, text_ids):
    tok = [TAGS[c - 1] if c else text_ids[p] for p, c in enumerate(classes)]
    n_checked = 0
    for outl, threads, endp, n_entries in blocks_of(classes):
        if len(threads) != n_entries:
            continue
        main = tok[:outl + 1]
        res = F.fork([main], TAGS, flags=F.FORK_SEED_ENTRY, lenient=True)
        assert res["status"] == [0] and res["worker_off"] == [0, n_entries]
        # seeds: the text between each entry's own tags, found by scanning the outline
        o = max(p for p in range(outl) if classes[p] == GP.OUT)
        seeds, p = [], o + 1
        while p < outl:
            if classes[p] in (GP.SUB, GP.TRI):
                q = p + 1
                while classes[q] == GP.TEXT:
                    q += 1
                seeds.append(tok[p + 1:q])
                p = q
            p += 1
        thr = TAGS[GP.THR - 1]
        assert res["ctx"] == [main + [thr] + sd for sd in seeds]
        seqs = [main + tok[a:b + 1] for a, b in threads]
        joined, st = F.join([main], res["worker_off"], seqs, TAGS)
        assert st == [0]
        # the join rebuilds the block without its gaps after </Outlines> and after threads
        inside = set()
        for a, b in threads:
            inside.update(range(a, b + 1))
        expect = main + [tok[x] for x in range(outl + 1, endp) if x in inside] + [tok[endp]]
        assert joined[0] == expect
        n_checked += 1
    return n_checked


def test_round_trip_lenient_streams():
    rng = random.Random(21)
    strings = [list(s) for s in GP.enumerate_valid(16, "lenient")]
    n = 0
    for s in rng.sample(strings, 3000):
        n += _round_trip_lenient(s, [rng.randrange(0, 99) for _ in s])
    assert n > 500


@pytest.mark.parametrize("names,strict,lenient", [
    ("think Par t Out Sub t /Sub /Out", F.ST_NO_OUTLINE, 0),
    ("think Par Out t Sub t /Sub /Out", F.ST_BAD_ENTRY, 0),
    ("think Par Out Sub t /Sub t t Tri t /Tri t /Out", F.ST_BAD_ENTRY, 0),
    ("think Par t t Out t Sub t t /Sub t /Out", F.ST_NO_OUTLINE, 0),
    ("think Par Out t /Out", F.ST_BAD_ENTRY, F.ST_BAD_ENTRY),
    ("think t Out Sub t /Sub /Out", F.ST_NO_OUTLINE, F.ST_NO_OUTLINE),
    ("think Thr t Out Sub t /Sub /Out", F.ST_NO_OUTLINE, F.ST_NO_OUTLINE),
    ("t t Out Sub t /Sub /Out", F.ST_NO_OUTLINE, F.ST_NO_OUTLINE),
    ("think Par Out Sub /Sub t /Out", F.ST_BAD_ENTRY, F.ST_BAD_ENTRY),
    ("think Par Out Sub t /Sub t Thr /Out", F.ST_BAD_ENTRY, F.ST_BAD_ENTRY),
])
def test_rows_strict_and_lenient(names, strict, lenient):
    row = toks(GP.parse_names(names))
    assert F.fork([row], TAGS)["status"] == [strict]
    assert F.fork([row], TAGS, lenient=True)["status"] == [lenient]
