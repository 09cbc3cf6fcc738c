"""Independent checkers used to pin the oracle (pure Python, tiny inputs only).

None of this code is shared with the oracle or the GPU library.  Each checker is
a textbook algorithm applied directly to the paper's definitions:

* ``earley`` -- an Earley recognizer run on the productions of the figure
  "Context-Free Grammar for Parason" (Sec. 3.2), extended by the reading that
  free text may follow </think>.  A prefix is viable exactly when its Earley set
  is non-empty (every non-terminal of the grammar is productive), which gives an
  independent first-error position.  ``grammar="lenient"`` adds a nullable
  ``Gap -> Text Gap | epsilon`` after <Parallel>, <Outlines>, every outline
  entry, </Outlines> and every thread (the line breaks of Figure 3).
* ``dag_latency`` -- builds the fork/join dependency DAG of a valid stream (each
  token waits for the previous token on its own path; the tokens of a block
  outside its threads form the block's own sequential chain, its threads fork
  after the last of them, and </Parallel> joins all threads) and takes the
  longest path, which is the "longest generation path" of Sec. 4
  ("Evaluation").
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
# The same grammar with optional Text runs between the structural tags of a
# parallel region.
LENIENT_GRAMMAR = dict(
    GRAMMAR,
    P=[[PAR, "Gap", "O", "Gap", "H", END_PAR]],
    O=[[OUT, "Gap", "G", END_OUT]],
    G=[["E", "Gap", "G"], ["E", "Gap"]],
    H=[["W", "Gap", "H"], ["W", "Gap"]],
    Gap=[[TEXT, "Gap"], []],
)
GRAMMARS = {"strict": GRAMMAR, "lenient": LENIENT_GRAMMAR}
START = "S0"


def _nullable(grammar):
    null = set()
    changed = True
    while changed:
        changed = False
        for a, alts in grammar.items():
            if a in null:
                continue
            for rhs in alts:
                if all(isinstance(s, str) and s in null for s in rhs):
                    null.add(a)
                    changed = True
                    break
    return null


NULLABLE = {name: _nullable(g) for name, g in GRAMMARS.items()}


def earley(classes, grammar="strict"):
    """Return (accepted, first_error_pos).

    first_error_pos is the length of the longest viable prefix when that prefix
    is shorter than the input; len(classes) when the whole input is viable but
    not a sentence (truncated); -1 when accepted.
    """
    GR = GRAMMARS[grammar]
    nullable = NULLABLE[grammar]
    n = len(classes)
    sets = [set() for _ in range(n + 1)]
    # item = (lhs, alt_index, dot, origin)

    def add(k, item, work):
        if item not in sets[k]:
            sets[k].add(item)
            work.append(item)

    work = []
    for ai in range(len(GR[START])):
        add(0, (START, ai, 0, 0), work)
    for k in range(n + 1):
        work = list(sets[k])
        while work:
            lhs, ai, dot, org = work.pop()
            rhs = GR[lhs][ai]
            if dot < len(rhs):
                sym = rhs[dot]
                if isinstance(sym, str):  # predict
                    for bi in range(len(GR[sym])):
                        add(k, (sym, bi, 0, k), work)
                    if sym in nullable:
                        add(k, (lhs, ai, dot + 1, org), work)
            else:  # complete
                for (l2, a2, d2, o2) in list(sets[org]):
                    r2 = GR[l2][a2]
                    if d2 < len(r2) and r2[d2] == lhs:
                        add(k, (l2, a2, d2 + 1, o2), work)
        if k == n:
            break
        tok = classes[k]
        for (lhs, ai, dot, org) in sets[k]:
            rhs = GR[lhs][ai]
            if dot < len(rhs) and rhs[dot] == tok:
                sets[k + 1].add((lhs, ai, dot + 1, org))
        if not sets[k + 1]:
            return False, k
    accepted = any(
        lhs == START and dot == len(GR[lhs][ai]) and org == 0
        for (lhs, ai, dot, org) in sets[n]
    )
    return (True, -1) if accepted else (False, n)


def dag_latency(classes):
    """Longest path (in tokens) through the fork/join DAG of a *valid* stream.

    Nodes are tokens, each costing 1.  Edges:
      * a token on a path (the root, a thread, or a block's own chain) waits
        for the previous token on that path;
      * a block's own chain is <Parallel> and every token of the block outside
        its threads except </Parallel> (the outline, and gap Text where the
        lenient grammar allows it); <Parallel> waits for the enclosing path;
      * every <Thread> of the block waits for the last token of that chain
        (the threads are dispatched once the main trajectory has decoded it);
      * </Parallel> waits for every </Thread> of the block, and the enclosing
        path continues from </Parallel>.
    Returns (latency, thread_latencies) where thread_latencies is a list with
    one list per block, in order of the block's </Parallel>, holding each
    thread's own longest path (from its <Thread> to its </Thread>).
    """
    n = len(classes)
    deps = [[] for _ in range(n)]
    fork_of = {}  # <Thread> index -> block id (resolved after the block closes)
    blocks = []  # open blocks: {"id", "chain_last", "ends", "starts"}
    paths = [None]  # per open path, the previous token on it; root first
    kinds = ["root"]  # "root", "block" or "thread" for each open path
    closed = {}
    finished = []
    bid = 0
    for i, c in enumerate(classes):
        if c == PAR:
            deps[i] = [paths[-1]]
            blocks.append({"id": bid, "chain_last": i, "ends": [], "starts": []})
            bid += 1
            paths.append(i)
            kinds.append("block")
        elif c == THR:
            b = blocks[-1]
            fork_of[i] = b["id"]
            b["starts"].append(i)
            paths.append(i)
            kinds.append("thread")
        elif c == END_THR:
            deps[i] = [paths[-1]]
            paths.pop()
            kinds.pop()
            blocks[-1]["ends"].append(i)
        elif c == END_PAR:
            b = blocks.pop()
            deps[i] = list(b["ends"])
            closed[b["id"]] = b["chain_last"]
            finished.append(b)
            paths.pop()
            kinds.pop()
            paths[-1] = i
            continue
        else:
            deps[i] = [paths[-1]]
            if kinds[-1] == "block":
                blocks[-1]["chain_last"] = i
        if c != END_THR:
            paths[-1] = i
    for t, b in fork_of.items():
        deps[t] = [closed[b]]
    dist = [None] * n

    def longest(i):
        stack = [i]
        while stack:
            j = stack[-1]
            if dist[j] is not None:
                stack.pop()
                continue
            todo = [d for d in deps[j] if d is not None and dist[d] is None]
            if todo:
                stack.extend(todo)
                continue
            dist[j] = 1 + max((dist[d] for d in deps[j] if d is not None), default=0)
            stack.pop()
        return dist[i]

    for i in range(n):
        longest(i)
    per_block = [[dist[e] - dist[s] + 1 for s, e in zip(b["starts"], b["ends"])] for b in finished]
    return (dist[-1] if classes else 0), per_block


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
def _gen(sym, maxlen, grammar):
    """All terminal strings (tuples) of length <= maxlen derivable from sym."""
    if maxlen < 0:
        return frozenset()
    if isinstance(sym, int):
        return frozenset([(sym,)]) if maxlen >= 1 else frozenset()
    res = set()
    for rhs in GRAMMARS[grammar][sym]:
        res |= _seq(tuple(rhs), maxlen, grammar)
    return frozenset(res)


@functools.lru_cache(maxsize=None)
def _seq(rhs, maxlen, grammar):
    if not rhs:
        return frozenset([()])
    head, rest = rhs[0], rhs[1:]
    # every symbol derives at least its minimal length; bound the head accordingly
    res = set()
    min_rest = sum(_minlen(s, grammar) for s in rest)
    for h in _gen(head, maxlen - min_rest, grammar):
        for r in _seq(rest, maxlen - len(h), grammar):
            res.add(h + r)
    return frozenset(res)


@functools.lru_cache(maxsize=None)
def _minlen(sym, grammar):
    if isinstance(sym, int):
        return 1
    best = None
    for rhs in GRAMMARS[grammar][sym]:
        if sym in rhs:  # skip directly recursive alternatives
            continue
        v = sum(_minlen(s, grammar) for s in rhs)
        best = v if best is None else min(best, v)
    return best


def enumerate_valid(maxlen, grammar="strict"):
    return sorted(_gen(START, maxlen, grammar), key=lambda s: (len(s), s))


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
