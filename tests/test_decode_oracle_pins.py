"""Pins of the decode-step oracle (CPU only).

The allowed next tokens after a prefix are fixed by the grammar of Figure 4
(Sec. 3.2) alone: a token may follow when the longer prefix can still be
completed to a valid stream.  The oracle gets them from the accounting parser;
these tests get them in two other ways -- an Earley recognizer on the grammar's
productions and brute force over every valid stream up to a length bound -- and
check a table of worked states written out from the grammar by hand."""
import random

import pytest

from oracle import decode_oracle as D
from oracle import oracle as O
from tests import grammar_pins as GP

TAGS = list(range(100, 112))
TEXT_ID = 7


def _toks(classes):
    return GP.to_tokens(classes, TAGS, TEXT_ID)


def _earley_allowed(classes):
    allowed = set()
    for c in range(13):
        ok, pos = GP.earley(classes + [c])
        if ok or pos == len(classes) + 1:
            allowed.add(c)
    return allowed, GP.earley(classes)[0]


# (prefix, allowed classes, eos allowed), read off the productions of Figure 4
WORKED = [
    ("", {GP.THINK}, False),
    ("think", {GP.TEXT, GP.PAR, GP.END_THINK}, False),
    ("think t3", {GP.TEXT, GP.PAR, GP.END_THINK}, False),
    ("think Par", {GP.OUT}, False),
    ("think Par Out", {GP.SUB, GP.TRI}, False),
    ("think Par Out Sub", {GP.TEXT}, False),
    ("think Par Out Tri t", {GP.TEXT, GP.END_TRI}, False),
    ("think Par Out Tri t /Tri", {GP.SUB, GP.TRI, GP.END_OUT}, False),
    ("think Par Out Sub t /Sub /Out", {GP.THR}, False),
    ("think Par Out Sub t /Sub /Out Thr", {GP.TEXT, GP.PAR, GP.END_THR}, False),
    ("think Par Out Sub t /Sub /Out Thr /Thr", {GP.THR, GP.END_PAR}, False),
    ("think Par Out Sub t /Sub /Out Thr Par Out Sub t /Sub /Out Thr t /Thr /Par",
     {GP.TEXT, GP.PAR, GP.END_THR}, False),
    ("think Par Out Sub t /Sub /Out Thr /Thr /Par", {GP.TEXT, GP.PAR, GP.END_THINK}, False),
    ("think /think", {GP.TEXT}, True),
    ("think t /think t2", {GP.TEXT}, True),
    # not viable any more: nothing may follow
    ("t", set(), False),
    ("think Par Out /Out", set(), False),
]


@pytest.mark.parametrize("prefix,allowed,eos", WORKED)
def test_worked_states(prefix, allowed, eos):
    got, got_eos = D.allowed_classes(_toks(GP.parse_names(prefix)), TAGS, TEXT_ID)
    assert got == allowed
    assert got_eos == eos


def test_matches_earley_on_random_walks():
    rng = random.Random(11)
    prefixes = []
    for _ in range(60):
        cls = []
        for _ in range(rng.randrange(0, 40)):
            allowed, _ = _earley_allowed(cls)
            if not allowed:
                break
            # favour tags so that walks reach nested blocks
            tags = sorted(allowed - {GP.TEXT})
            cls.append(rng.choice(tags) if tags and rng.random() < 0.7 else rng.choice(sorted(allowed)))
        prefixes.append(cls)
        # and one token that breaks the prefix, when there is one
        bad = sorted(set(range(13)) - _earley_allowed(cls)[0])
        if bad:
            prefixes.append(cls + [rng.choice(bad)])
    got = D.allowed_batch([_toks(p) for p in prefixes], TAGS, TEXT_ID)
    for p, g in zip(prefixes, got):
        assert g == _earley_allowed(p), GP.NAMES and [GP.NAMES[c] for c in p]
        assert g == D.allowed_classes(_toks(p), TAGS, TEXT_ID)


def test_matches_brute_force_over_short_streams():
    maxlen = 13
    valid = GP.enumerate_valid(maxlen)
    nxt = {}
    for s in valid:
        for k in range(len(s)):
            nxt.setdefault(s[:k], set()).add(s[k])
    complete = set(valid)
    # allowed must contain every continuation seen; for prefixes short enough
    # that every allowed continuation completes within maxlen, it is exactly that
    prefixes = sorted(nxt, key=lambda p: (len(p), p))
    got = D.allowed_batch([_toks(list(p)) for p in prefixes], TAGS, TEXT_ID)
    exact = 0
    for p, (allowed, eos) in zip(prefixes, got):
        assert nxt[p] <= allowed
        assert eos == (p in complete)
        if len(p) <= 3:  # the longest shortest completion of an allowed token is 10
            assert allowed == nxt[p], [GP.NAMES[c] for c in p]
            exact += 1
    assert exact >= 10


def test_eos_never_before_end_think():
    assert D.allowed_classes([], TAGS, TEXT_ID)[1] is False
    assert D.allowed_classes(_toks(GP.parse_names("think t")), TAGS, TEXT_ID)[1] is False


# --------------------------------------------------------------------------- lenient gaps

LENIENT = O.CFG_LENIENT_GAPS

# with the lenient-gaps reading Text joins the allowed set between a region's
# structural tags, and leaves every other state as it was
WORKED_LENIENT = [
    ("", {GP.THINK}, False),
    ("think", {GP.TEXT, GP.PAR, GP.END_THINK}, False),
    ("think Par", {GP.TEXT, GP.OUT}, False),
    ("think Par t2", {GP.TEXT, GP.OUT}, False),
    ("think Par t Out", {GP.TEXT, GP.SUB, GP.TRI}, False),
    ("think Par Out Sub", {GP.TEXT}, False),
    ("think Par Out Tri t", {GP.TEXT, GP.END_TRI}, False),
    ("think Par Out Tri t /Tri", {GP.TEXT, GP.SUB, GP.TRI, GP.END_OUT}, False),
    ("think Par Out Tri t /Tri t", {GP.TEXT, GP.SUB, GP.TRI, GP.END_OUT}, False),
    ("think Par Out Sub t /Sub /Out", {GP.TEXT, GP.THR}, False),
    ("think Par Out Sub t /Sub /Out t", {GP.TEXT, GP.THR}, False),
    ("think Par Out Sub t /Sub /Out Thr", {GP.TEXT, GP.PAR, GP.END_THR}, False),
    ("think Par Out Sub t /Sub /Out Thr /Thr", {GP.TEXT, GP.THR, GP.END_PAR}, False),
    ("think Par Out Sub t /Sub /Out Thr /Thr t3", {GP.TEXT, GP.THR, GP.END_PAR}, False),
    ("think Par Out Sub t /Sub /Out Thr /Thr /Par", {GP.TEXT, GP.PAR, GP.END_THINK}, False),
    ("think /think", {GP.TEXT}, True),
    ("t", set(), False),
    ("think Par Out t /Out", set(), False),
]


@pytest.mark.parametrize("prefix,allowed,eos", WORKED_LENIENT)
def test_worked_states_lenient(prefix, allowed, eos):
    got, got_eos = D.allowed_classes(_toks(GP.parse_names(prefix)), TAGS, TEXT_ID, LENIENT)
    assert got == allowed
    assert got_eos == eos


def _earley_allowed_lenient(classes):
    allowed = set()
    for c in range(13):
        ok, pos = GP.earley(classes + [c], "lenient")
        if ok or pos == len(classes) + 1:
            allowed.add(c)
    return allowed, GP.earley(classes, "lenient")[0]


def test_lenient_matches_earley_on_random_walks():
    rng = random.Random(12)
    prefixes = []
    for _ in range(60):
        cls = []
        for _ in range(rng.randrange(0, 40)):
            allowed, _ = _earley_allowed_lenient(cls)
            if not allowed:
                break
            tags = sorted(allowed - {GP.TEXT})
            cls.append(rng.choice(tags) if tags and rng.random() < 0.6 else rng.choice(sorted(allowed)))
        prefixes.append(cls)
        bad = sorted(set(range(13)) - _earley_allowed_lenient(cls)[0])
        if bad:
            prefixes.append(cls + [rng.choice(bad)])
    got = D.allowed_batch([_toks(p) for p in prefixes], TAGS, TEXT_ID, LENIENT)
    for p, g in zip(prefixes, got):
        assert g == _earley_allowed_lenient(p), [GP.NAMES[c] for c in p]
