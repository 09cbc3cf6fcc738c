"""Independent checkers used to pin the oracle (pure Python, tiny inputs only).

None of this code is shared with the oracle or the GPU library.  Each checker is
a textbook algorithm applied directly to the paper's definitions:

* ``earley`` -- an Earley recognizer run on the productions of the figure
  "Context-Free Grammar for Parason" (Sec. 3.2), extended by the reading that
  free text may follow </think>.  A prefix is viable exactly when its Earley set
  is non-empty (every non-terminal of the grammar is productive), which gives an
  independent first-error position.
* ``dag_latency`` -- builds the fork/join dependency DAG of a valid stream (each
  token waits for the previous token on its own path; the threads of a block
  fork after </Outlines> and </Parallel> joins all of them) and takes the longest
  path, which is the "longest generation path" of Sec. 4 ("Evaluation").
* ``enumerate_valid`` -- grammar-directed enumeration of every valid class
  string up to a length bound.

Class codes: 0 = Text, 1..12 = the tags in the order
<think> </think> <Parallel> </Parallel> <Outlines> </Outlines>
<Subtask> </Subtask> <Trial> </Trial> <Thread> </Thread>.
"""
from __future__ import annotations

import functools

TEXT, THINK, END_THINK, PAR, END_PAR, OUT, END_OUT, SUB, END_SUB, TRI, END_TRI, THR, END_THR = range(13)
NAMES = ["t", "think", "/think", "Par", "/Par", "Out", "/Out", "Sub", "/Sub", "Tri", "/Tri", "Thr", "/Thr"]
BY_NAME = {n: i for i, n in enumerate(NAMES)}

# Productions.  Upper-case strings are non-terminals, ints are terminals.
GRAMMAR = {
    "S0": [["S", "Tail"]],
    "Tail": [[TEXT, "Tail"], []],
    "S": [[THINK, "B", END_THINK]],
    "B": [["T", "B"], ["P", "B"], []],
    "P": [[PAR, "O", "H", END_PAR]],
    "O": [[OUT, "G", END_OUT]],
    "G": [["E", "G"], ["E"]],
    "E": [[SUB, "T", END_SUB], [TRI, "T", END_TRI]],
    "H": [["W", "H"], ["W"]],
    "W": [[THR, "B", END_THR]],
    "T": [[TEXT, "T"], [TEXT]],
}
START = "S0"


def _nullable():
    null = set()
    changed = True
    while changed:
        changed = False
        for a, alts in GRAMMAR.items():
            if a in null:
                continue
            for rhs in alts:
                if all(isinstance(s, str) and s in null for s in rhs):
                    null.add(a)
                    changed = True
                    break
    return null


NULLABLE = _nullable()


def earley(classes):
    """Return (accepted, first_error_pos).

    first_error_pos is the length of the longest viable prefix when that prefix
    is shorter than the input; len(classes) when the whole input is viable but
    not a sentence (truncated); -1 when accepted.
    """
    n = len(classes)
    sets = [set() for _ in range(n + 1)]
    # item = (lhs, alt_index, dot, origin)

    def add(k, item, work):
        if item not in sets[k]:
            sets[k].add(item)
            work.append(item)

    work = []
    for ai in range(len(GRAMMAR[START])):
        add(0, (START, ai, 0, 0), work)
    for k in range(n + 1):
        work = list(sets[k])
        while work:
            lhs, ai, dot, org = work.pop()
            rhs = GRAMMAR[lhs][ai]
            if dot < len(rhs):
                sym = rhs[dot]
                if isinstance(sym, str):  # predict
                    for bi in range(len(GRAMMAR[sym])):
                        add(k, (sym, bi, 0, k), work)
                    if sym in NULLABLE:
                        add(k, (lhs, ai, dot + 1, org), work)
            else:  # complete
                for (l2, a2, d2, o2) in list(sets[org]):
                    r2 = GRAMMAR[l2][a2]
                    if d2 < len(r2) and r2[d2] == lhs:
                        add(k, (l2, a2, d2 + 1, o2), work)
        if k == n:
            break
        tok = classes[k]
        for (lhs, ai, dot, org) in sets[k]:
            rhs = GRAMMAR[lhs][ai]
            if dot < len(rhs) and rhs[dot] == tok:
                sets[k + 1].add((lhs, ai, dot + 1, org))
        if not sets[k + 1]:
            return False, k
    accepted = any(
        lhs == START and dot == len(GRAMMAR[lhs][ai]) and org == 0
        for (lhs, ai, dot, org) in sets[n]
    )
    return (True, -1) if accepted else (False, n)


def dag_latency(classes):
    """Longest path (in tokens) through the fork/join DAG of a *valid* stream.

    Returns (latency, thread_latencies) where thread_latencies is a list with
    one list per block, in order of the block's </Parallel>, holding each
    thread's own longest path (from its <Thread> to its </Thread>).
    """
    dist = [0] * len(classes)
    blocks = []  # stack of dicts: fork node, thread end nodes, thread start nodes
    finished = []
    pred = None
    for i, c in enumerate(classes):
        if c == PAR:
            deps = [pred]
            blocks.append({"fork": None, "ends": [], "starts": []})
        elif c == END_OUT:
            deps = [pred]
            blocks[-1]["fork"] = i
        elif c == THR:
            deps = [blocks[-1]["fork"]]
            blocks[-1]["starts"].append(i)
        elif c == END_THR:
            deps = [pred]
            blocks[-1]["ends"].append(i)
        elif c == END_PAR:
            deps = blocks[-1]["ends"]
            b = blocks.pop()
            finished.append([dist[e] - dist[s] + 1 for s, e in zip(b["starts"], b["ends"])])
        else:
            deps = [pred]
        base = max((dist[d] for d in deps if d is not None), default=0)
        dist[i] = base + 1
        pred = i if c != END_THR else None
    return (dist[-1] if classes else 0), finished


def thread_types(classes):
    """Branch type (0 main, 1 Subtask, 2 Trial) of the innermost enclosing thread
    of every token of a *valid* stream, via an explicit bracket stack.  Thread k
    of a block pairs with outline entry k; surplus threads are untyped (0)."""
    out = []
    stack = []  # per open block: {"entries": [...], "k": next thread index, "cur": type of open thread}
    ctx = [0]  # type stack: innermost open thread type at the end
    for c in classes:
        if c == PAR:
            stack.append({"entries": [], "k": 0})
            out.append(ctx[-1])
        elif c in (SUB, TRI) and stack:
            stack[-1]["entries"].append(1 if c == SUB else 2)
            out.append(ctx[-1])
        elif c == THR:
            b = stack[-1]
            t = b["entries"][b["k"]] if b["k"] < len(b["entries"]) else 0
            b["k"] += 1
            ctx.append(t)
            out.append(t)
        elif c == END_THR:
            out.append(ctx.pop())
        elif c == END_PAR:
            stack.pop()
            out.append(ctx[-1])
        else:
            out.append(ctx[-1])
    return out


@functools.lru_cache(maxsize=None)
def _gen(sym, maxlen):
    """All terminal strings (tuples) of length <= maxlen derivable from sym."""
    if maxlen < 0:
        return frozenset()
    if isinstance(sym, int):
        return frozenset([(sym,)]) if maxlen >= 1 else frozenset()
    res = set()
    for rhs in GRAMMAR[sym]:
        res |= _seq(tuple(rhs), maxlen)
    return frozenset(res)


@functools.lru_cache(maxsize=None)
def _seq(rhs, maxlen):
    if not rhs:
        return frozenset([()])
    head, rest = rhs[0], rhs[1:]
    # every symbol derives at least its minimal length; bound the head accordingly
    res = set()
    min_rest = sum(_minlen(s) for s in rest)
    for h in _gen(head, maxlen - min_rest):
        for r in _seq(rest, maxlen - len(h)):
            res.add(h + r)
    return frozenset(res)


@functools.lru_cache(maxsize=None)
def _minlen(sym):
    if isinstance(sym, int):
        return 1
    best = None
    for rhs in GRAMMAR[sym]:
        if sym in rhs:  # skip directly recursive alternatives
            continue
        v = sum(_minlen(s) for s in rhs)
        best = v if best is None else min(best, v)
    return best


def enumerate_valid(maxlen):
    return sorted(_gen(START, maxlen), key=lambda s: (len(s), s))


def parse_names(text):
    """'think t t Par ...' -> class list; 'tN' expands to N Text tokens."""
    out = []
    for w in text.split():
        if w in BY_NAME:
            out.append(BY_NAME[w])
        elif w.startswith("t") and w[1:].isdigit():
            out.extend([TEXT] * int(w[1:]))
        else:
            raise ValueError(w)
    return out


def to_tokens(classes, tag_ids, text_id=7):
    """Class string -> token ids (Text uses text_id, which must not be a tag)."""
    assert text_id not in set(tag_ids)
    return [text_id if c == TEXT else int(tag_ids[c - 1]) for c in classes]
