"""Pins of the oracle's lenient mode (CFG_LENIENT_GAPS).

Figure 3 lays a parallel region out with line breaks between its structural
tags, which the grammar of Figure 4 as printed does not allow.  In lenient mode
a run of Text may follow <Parallel>, <Outlines>, every outline entry,
</Outlines> and every </Thread> of a region.  Those tokens are decoded by the
enclosing path, like the outline, so they lengthen the block's sequential part
and take the enclosing branch type.

Every check compares the oracle with something other than itself: an Earley
recognizer on the lenient productions, the fork/join DAG longest path, a tree
evaluator, the strict grammar (a lenient stream without gaps is a strict
stream; moving a block's gaps into its first entry's text gives a strict
stream with the same accounting), and a hand-computed golden.
"""
import json
import os
import random

import numpy as np
import pytest

import grammar_pins as G
from oracle import oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
TAGS = np.arange(151936 - 12, 151936, dtype=np.int32)
SCATTERED = np.array([5, 900, 17, 151000, 3, 77777, 42, 1000, 2**31 - 1, 123456, 64, 8], dtype=np.int32)
LENIENT = O.CFG_LENIENT_GAPS


def run(classes, tags=TAGS, flags=LENIENT):
    return O.eval_stream(G.to_tokens(classes, tags, 7), tags, flags)


def run_many(streams, tags=TAGS, flags=LENIENT):
    toks = np.concatenate([np.array(G.to_tokens(s, tags, 7), np.int32) for s in streams] + [np.zeros(1, np.int32)])
    lens = np.array([len(s) for s in streams], np.int32)
    starts = np.concatenate([[0], np.cumsum(lens)[:-1]]).astype(np.int64)
    return O.eval_rows(toks, starts, lens, tags, flags)


def independent_row(classes):
    lat, _ = G.dag_latency(classes)
    types = G.thread_types(classes)
    d = m = 0
    for c in classes:
        if c == G.PAR:
            d += 1
            m = max(m, d)
        elif c == G.END_PAR:
            d -= 1
    return dict(total=len(classes), latency=lat, n_subtask=types.count(1), n_trial=types.count(2),
                n_blocks=classes.count(G.PAR), max_depth=m)


def check_row(r, classes):
    for k, v in independent_row(classes).items():
        assert int(r[k]) == v, (k, int(r[k]), v, " ".join(G.NAMES[c] for c in classes))


FIELDS = ("total", "latency", "n_subtask", "n_trial", "n_blocks", "max_depth", "first_error_pos", "flags")


# --------------------------------------------------------------------------- language


@pytest.mark.parametrize("tags", [TAGS, SCATTERED], ids=["contiguous", "scattered"])
def test_every_valid_lenient_string_up_to_17(tags):
    strings = [list(s) for s in G.enumerate_valid(17, "lenient")]
    assert len(strings) > 20000
    rows = run_many(strings, tags)
    for s, r in zip(strings, rows):
        assert r["flags"] & O.F_VALID and r["first_error_pos"] == -1, s
        check_row(r, s)


def test_strict_streams_are_unchanged_in_lenient_mode():
    strings = [list(s) for s in G.enumerate_valid(18)]
    strict = run_many(strings, flags=0)
    lenient = run_many(strings)
    for k in FIELDS:
        assert np.array_equal(strict[k], lenient[k]), k


def test_gap_streams_are_rejected_in_strict_mode_at_the_first_gap():
    strings = [list(s) for s in G.enumerate_valid(16, "lenient")]
    strict_set = set(map(tuple, G.enumerate_valid(16)))
    gap_strings = [s for s in strings if tuple(s) not in strict_set]
    assert len(gap_strings) > 5000
    rows = run_many(gap_strings, flags=0)
    for s, r in zip(gap_strings, rows):
        ok, err = G.earley(s, "strict")
        assert not ok
        assert not (r["flags"] & O.F_VALID) and int(r["first_error_pos"]) == err
        assert s[err] == G.TEXT  # the first gap token breaks the strict grammar


def _mutations(s, rng, k):
    out = []
    n = len(s)
    for _ in range(k):
        op = rng.randrange(4)
        if op == 0 and n:
            i = rng.randrange(n)
            out.append(s[:i] + [rng.randrange(13)] + s[i + 1:])
        elif op == 1 and n:
            i = rng.randrange(n)
            out.append(s[:i] + s[i + 1:])
        elif op == 2:
            i = rng.randrange(n + 1)
            out.append(s[:i] + [G.TEXT] * rng.randint(1, 3) + s[i:])  # a Text run anywhere
        else:
            i = rng.randrange(n + 1)
            out.append(s[:i] + [rng.randrange(13)] + s[i:])
    return out


def test_lenient_validity_and_first_error_match_earley():
    rng = random.Random(77)
    strings = [list(s) for s in G.enumerate_valid(17, "lenient")]
    cases = []
    for s in rng.sample(strings, 1500):
        cases += _mutations(s, rng, 4)
        cases.append(s[: rng.randrange(len(s) + 1)])
    rows = run_many(cases)
    n_invalid = 0
    for s, r in zip(cases, rows):
        ok, err = G.earley(s, "lenient")
        assert bool(r["flags"] & O.F_VALID) == ok, s
        assert int(r["first_error_pos"]) == err, (s, int(r["first_error_pos"]), err)
        assert bool(r["flags"] & O.F_TRUNCATED) == (not ok and err == len(s))
        if ok:
            check_row(r, s)
        else:
            n_invalid += 1
            assert (r["latency"], r["n_subtask"], r["n_trial"], r["n_blocks"], r["max_depth"]) == (len(s), 0, 0, 0, 0)
    assert n_invalid > 2000


def test_lenient_random_short_strings_match_earley():
    rng = random.Random(4242)
    weights = [6] + [1] * 12  # Text more often, so gaps appear
    cases = []
    for _ in range(20000):
        n = rng.randrange(0, 10)
        body = rng.choices(range(13), weights=weights, k=n)
        cases.append([G.THINK, G.PAR] + body if rng.random() < 0.7 else body)
    rows = run_many(cases)
    for s, r in zip(cases, rows):
        ok, err = G.earley(s, "lenient")
        assert bool(r["flags"] & O.F_VALID) == ok, s
        assert int(r["first_error_pos"]) == err, s


def test_text_before_think_stays_invalid():
    r = run([G.TEXT, G.THINK, G.END_THINK])
    assert r["flags"] == 0 and r["first_error_pos"] == 0
    # an entry still needs text of its own: a gap does not fill it
    s = G.parse_names("think Par Out t2 Sub /Sub")
    r = run(s)
    assert r["flags"] == 0 and r["first_error_pos"] == 6  # the empty entry closes at 6


# --------------------------------------------------------------------------- closed forms and trees


def test_lenient_single_block_closed_form():
    rng = random.Random(8)
    for _ in range(300):
        k = rng.randint(1, 5)
        entries = [rng.randint(1, 6) for _ in range(k)]
        bodies = [rng.randint(0, 30) for _ in range(k)]
        g_par, g_out, g_close = rng.randint(0, 3), rng.randint(0, 3), rng.randint(0, 3)
        g_entry = [rng.randint(0, 3) for _ in range(k)]
        g_thread = [rng.randint(0, 3) for _ in range(k)]
        a, b = rng.randint(0, 9), rng.randint(0, 9)
        kind = rng.choice([G.SUB, G.TRI])
        close = G.END_SUB if kind == G.SUB else G.END_TRI
        s = [G.THINK] + [G.TEXT] * a + [G.PAR] + [G.TEXT] * g_par + [G.OUT] + [G.TEXT] * g_out
        for e, g in zip(entries, g_entry):
            s += [kind] + [G.TEXT] * e + [close] + [G.TEXT] * g
        s += [G.END_OUT] + [G.TEXT] * g_close
        for x, g in zip(bodies, g_thread):
            s += [G.THR] + [G.TEXT] * x + [G.END_THR] + [G.TEXT] * g
        s += [G.END_PAR] + [G.TEXT] * b + [G.END_THINK]
        r = run(s)
        gaps = g_par + g_out + g_close + sum(g_entry) + sum(g_thread)
        lat = (a + b) + 2 + 2 + (2 + sum(2 + e for e in entries)) + gaps + max(2 + x for x in bodies)
        assert r["flags"] & O.F_VALID
        assert r["latency"] == lat and r["total"] == len(s)
        branch = sum(2 + x for x in bodies)
        assert r["n_subtask" if kind == G.SUB else "n_trial"] == branch  # gaps are main-path tokens
        assert r["total"] - r["latency"] == branch - max(2 + x for x in bodies)


def random_body(rng, depth, budget):
    items = []
    for _ in range(rng.randint(0, 3)):
        if depth < 4 and rng.random() < 0.45:
            items.append(random_block(rng, depth + 1, budget))
        else:
            items.append(rng.randint(1, budget))
    return items


def random_block(rng, depth, budget):
    n_e = rng.randint(1, 4)
    n_t = n_e if rng.random() < 0.85 else rng.randint(1, 5)
    entries = [(rng.choice([G.SUB, G.TRI]), rng.randint(1, budget)) for _ in range(n_e)]
    threads = [random_body(rng, depth, budget) for _ in range(n_t)]
    gap = lambda: rng.choice([0, 0, 1, 1, 2, 5])  # noqa: E731
    gaps = dict(par=gap(), out=gap(), close=gap(), entry=[gap() for _ in entries], thread=[gap() for _ in threads])
    return ("P", entries, threads, gaps)


def render(items, out, with_gaps=True):
    """Render a tree.  Without gaps, every block's gap tokens are moved into the
    text of its first outline entry (a strict stream)."""
    for it in items:
        if isinstance(it, int):
            out += [G.TEXT] * it
            continue
        _, entries, threads, g = it
        total_gap = g["par"] + g["out"] + g["close"] + sum(g["entry"]) + sum(g["thread"])
        gp = (lambda n: [G.TEXT] * n) if with_gaps else (lambda n: [])
        out += [G.PAR] + gp(g["par"]) + [G.OUT] + gp(g["out"])
        for j, (kind, e) in enumerate(entries):
            extra = total_gap if (j == 0 and not with_gaps) else 0
            out += [kind] + [G.TEXT] * (e + extra) + [G.END_SUB if kind == G.SUB else G.END_TRI] + gp(g["entry"][j])
        out += [G.END_OUT] + gp(g["close"])
        for t, gt in zip(threads, g["thread"]):
            out.append(G.THR)
            render(t, out, with_gaps)
            out.append(G.END_THR)
            out += gp(gt)
        out.append(G.END_PAR)
    return out


def tree_eval(items, ctx, counts):
    """Latency of a body by structural recursion over the tree; counts[ctx]
    collects the tokens of each branch type (0 main, 1 Subtask, 2 Trial)."""
    lat = 0
    for it in items:
        if isinstance(it, int):
            lat += it
            counts[ctx] += it
            continue
        _, entries, threads, g = it
        seq = 1 + g["par"] + 1 + g["out"] + sum(2 + e + ge for (_, e), ge in zip(entries, g["entry"]))
        seq += 1 + g["close"] + sum(g["thread"])
        counts[ctx] += seq + 1  # the block's own tokens, </Parallel> included
        longest = 0
        for k, t in enumerate(threads):
            typ = (1 if entries[k][0] == G.SUB else 2) if k < len(entries) else 0
            counts[typ] += 2
            longest = max(longest, 2 + tree_eval(t, typ, counts))
        lat += seq + longest + 1
    return lat


def test_lenient_random_trees():
    rng = random.Random(31337)
    trees, lenient_streams, strict_streams = [], [], []
    for _ in range(400):
        body = random_body(rng, 0, 9)
        tail = rng.randint(0, 4)
        trees.append(body)
        lenient_streams.append([G.THINK] + render(body, []) + [G.END_THINK] + [G.TEXT] * tail)
        strict_streams.append([G.THINK] + render(body, [], with_gaps=False) + [G.END_THINK] + [G.TEXT] * tail)
    rl = run_many(lenient_streams)
    rs = run_many(strict_streams, flags=0)
    for body, s, a, b in zip(trees, lenient_streams, rl, rs):
        assert a["flags"] & O.F_VALID, s
        check_row(a, s)
        counts = [0, 0, 0]
        lat = 2 + tree_eval(body, 0, counts) + (len(s) - 1 - s.index(G.END_THINK))
        assert a["latency"] == lat
        assert (a["n_subtask"], a["n_trial"]) == (counts[1], counts[2])
        # moving each block's gaps into its first entry's text leaves every count unchanged
        for k in ("total", "latency", "n_subtask", "n_trial", "n_blocks", "max_depth", "flags"):
            assert a[k] == b[k], k
    assert sum(1 for s, t in zip(lenient_streams, strict_streams) if s != t) > 150  # rows with gaps


def test_repaired_figure3_with_line_breaks_golden():
    g = json.load(open(os.path.join(GOLDEN, "fig3_repaired_line_breaks.json")))
    s = G.parse_names(g["stream"])
    ok, _ = G.earley(s, "lenient")
    assert ok and not G.earley(s, "strict")[0]
    for tags in (TAGS, SCATTERED):
        r = run(s, tags)
        for k, v in g["expected"].items():
            assert int(r[k]) == v, (k, int(r[k]), v)
    for k, v in independent_row(s).items():
        assert g["expected"][k] == v
    # without the line breaks it is the strict golden
    strict = json.load(open(os.path.join(GOLDEN, "fig3_repaired.json")))
    assert G.parse_names(strict["stream"]) == _strip_gaps(s, g["line_break_tokens"])


def _strip_gaps(s, gap_len):
    """Remove the gap_len Text tokens after each tag that opens a gap in a
    parallel region (<Parallel>, <Outlines>, entry closes, </Outlines>,
    </Thread> when followed by more of the region)."""
    out = []
    i = 0
    openers = {G.PAR, G.OUT, G.END_SUB, G.END_TRI, G.END_OUT, G.END_THR}
    while i < len(s):
        out.append(s[i])
        if s[i] in openers and i + gap_len < len(s) and all(c == G.TEXT for c in s[i + 1:i + 1 + gap_len]):
            i += 1 + gap_len
        else:
            i += 1
    return out
