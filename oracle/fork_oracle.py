"""CPU oracle of fork/join packing for tool-call execution.

TEST INFRASTRUCTURE.  Only the tests, smoke() and the CPU baseline of bench.py
may import this module.

At inference the runtime decodes a trajectory until a <Parallel> region's
outline is complete, dispatches every <Subtask> / <Trial> entry of that outline
as an independent worker, and returns the workers' <Thread> outputs to the
main trajectory (Sec. 3.4, "Inference"; format of Figure 4, Sec. 3.2).  The
paper leaves the token-level packing open; this module fixes it as follows
(the same readings bind the GPU path):

fork
    A main row must end with </Outlines>.  Its outline is the region from the
    last <Outlines> before that end, which must directly follow a <Parallel>,
    and must hold one or more entries <Subtask> text+ </Subtask> or
    <Trial> text+ </Trial> back to back.  With ``lenient`` (the lenient-gaps
    reading of the grammar) Text may stand between <Parallel> and <Outlines>,
    after <Outlines>, between entries and before </Outlines>; the seed is still
    the entry's own text.  Worker k of the row gets the context
        row ++ [<Thread>] ++ (text of entry k, if seeding)
    Workers are numbered row by row, entry by entry; worker_off[i] is the
    first worker of row i.  A row whose outline breaks these rules gets no
    worker and a status bit.

join
    Worker w of row i returns its whole sequence: its context followed by what
    it generated, ending with its </Thread>.  The joined row is
        row ++ seq_w[len(row):] for the row's workers in order
            ++ [</Parallel>] (if closing)
    i.e. every worker contributes its own <Thread> ... </Thread> span exactly
    as it saw it.  With append-only, the row itself is left out (the caller
    appends in place).  A worker sequence that does not continue with
    <Thread> right after the row, or does not end with </Thread>, is copied
    as it is and flags its row.
"""
from __future__ import annotations

import numpy as np

THINK, END_THINK, PAR, END_PAR, OUT, END_OUT, SUB, END_SUB, TRI, END_TRI, THR, END_THR = range(1, 13)

FORK_SEED_ENTRY = 1 << 0
JOIN_CLOSE_PARALLEL = 1 << 0
JOIN_APPEND_ONLY = 1 << 1

ST_NO_OUTLINE_END = 1 << 0   # the row does not end with </Outlines>
ST_NO_OUTLINE = 1 << 1       # no <Outlines> before it, or not right after <Parallel>
ST_BAD_ENTRY = 1 << 2        # the region is not a sequence of well-formed entries
ST_BAD_THREAD = 1 << 3       # join: a worker sequence is not <Thread> ... </Thread> after the row


def _classes(row, tag_ids):
    cls = {int(t): k + 1 for k, t in enumerate(tag_ids)}
    return [cls.get(int(t), 0) for t in row]


def parse_outline(row, tag_ids, lenient=False):
    """(status, entries) of a main row; entries = [(kind, text_start, text_end)]
    with kind SUB or TRI and the entry's text at row[text_start:text_end]."""
    c = _classes(row, tag_ids)
    L = len(c)
    if L == 0 or c[-1] != END_OUT:
        return ST_NO_OUTLINE_END, []
    o = L - 2
    while o >= 0 and c[o] != OUT:
        o -= 1
    q = o - 1  # the token that must be <Parallel>
    while lenient and q >= 0 and c[q] == 0:
        q -= 1
    if o < 0 or q < 0 or c[q] != PAR:
        return ST_NO_OUTLINE, []
    entries = []
    p = o + 1
    while p < L - 1:
        while lenient and p < L - 1 and c[p] == 0:  # a gap
            p += 1
        if p == L - 1:
            break
        if c[p] not in (SUB, TRI):
            return ST_BAD_ENTRY, []
        q = p + 1
        while q < L - 1 and c[q] == 0:
            q += 1
        if q == L - 1 or c[q] != c[p] + 1 or q == p + 1:
            return ST_BAD_ENTRY, []
        entries.append((c[p], p + 1, q))
        p = q + 1
    if not entries:
        return ST_BAD_ENTRY, []
    return 0, entries


def fork(rows, tag_ids, flags=FORK_SEED_ENTRY, lenient=False):
    """rows: list of int sequences.  Returns dict with per-row status and
    worker_off (n + 1), and per-worker context (list of lists), row, entry index,
    kind."""
    thread = int(tag_ids[THR - 1])
    status, off = [], [0]
    ctx, w_row, w_entry, w_kind = [], [], [], []
    for i, row in enumerate(rows):
        row = [int(t) for t in row]
        st, entries = parse_outline(row, tag_ids, lenient)
        status.append(st)
        for k, (kind, a, b) in enumerate(entries):
            seed = row[a:b] if flags & FORK_SEED_ENTRY else []
            ctx.append(row + [thread] + seed)
            w_row.append(i)
            w_entry.append(k)
            w_kind.append(kind)
        off.append(off[-1] + len(entries))
    return dict(status=status, worker_off=off, ctx=ctx, row=w_row, entry=w_entry, kind=w_kind)


def join(rows, worker_off, worker_seqs, tag_ids, flags=JOIN_CLOSE_PARALLEL):
    """Joined rows and per-row status (ST_BAD_THREAD)."""
    thread, end_thread, end_par = (int(tag_ids[THR - 1]), int(tag_ids[END_THR - 1]), int(tag_ids[END_PAR - 1]))
    out, status = [], []
    for i, row in enumerate(rows):
        row = [int(t) for t in row]
        L = len(row)
        res = [] if flags & JOIN_APPEND_ONLY else list(row)
        st = 0
        for w in range(worker_off[i], worker_off[i + 1]):
            seq = [int(t) for t in worker_seqs[w]]
            tail = seq[L:]
            if len(tail) < 2 or tail[0] != thread or tail[-1] != end_thread:
                st |= ST_BAD_THREAD
            res += tail
        if flags & JOIN_CLOSE_PARALLEL:
            res.append(end_par)
        out.append(res)
        status.append(st)
    return out, status


def pack(rows):
    """Packed (tokens, starts, lengths) numpy arrays of a list of rows."""
    lengths = np.array([len(r) for r in rows], dtype=np.int32)
    starts = np.zeros(len(rows), dtype=np.int64)
    if len(rows):
        starts[1:] = np.cumsum(lengths[:-1].astype(np.int64))
    tokens = np.array([t for r in rows for t in r] or [], dtype=np.int32)
    return tokens, starts, lengths
