"""Hand-built token streams for parity tests (shared by the GPU tests and the
CPU emulation tests): every short valid string of the grammar of Figure 4
(Sec. 3.2) and mutations of them, nesting across the automaton's tiers,
outlines beyond the fast path's entry count, all-tag rows, tags straddling
segment boundaries and the repaired Figure 3."""
import json
import os

import numpy as np

import grammar_pins as GP

G = 8


def pack(streams, tags, text_ids=None):
    """Class strings -> packed tokens, starts, lengths (rows padded to a multiple of G)."""
    rng = np.random.default_rng(len(streams))
    toks = []
    for s in streams:
        t = np.array(GP.to_tokens(s, tags), dtype=np.int32) if len(s) else np.zeros(0, np.int32)
        if text_ids is None:
            text = rng.integers(0, 150000, size=t.size).astype(np.int32)
        else:
            text = rng.choice(np.asarray(text_ids, np.int32), size=t.size)
        text = np.where(np.isin(text, tags), 7, text)
        is_text = np.array([c == GP.TEXT for c in s], dtype=bool) if len(s) else np.zeros(0, bool)
        toks.append(np.where(is_text, text, t))
    while len(toks) % G:
        toks.append(np.array(GP.to_tokens(GP.parse_names("think t3 /think"), tags), np.int32))
    lengths = np.array([t.size for t in toks], np.int32)
    starts = np.zeros(len(toks), np.int64)
    starts[1:] = np.cumsum(lengths[:-1])
    tokens = np.concatenate(toks) if lengths.sum() else np.zeros(0, np.int32)
    return tokens, starts, lengths


def deep_stream(depth, kind=GP.SUB):
    close = GP.END_SUB if kind == GP.SUB else GP.END_TRI
    s = [GP.THINK]
    for _ in range(depth):
        s += [GP.PAR, GP.OUT, kind, GP.TEXT, close, GP.END_OUT, GP.THR, GP.TEXT]
    for _ in range(depth):
        s += [GP.END_THR, GP.END_PAR]
    return s + [GP.END_THINK]


def fanout_stream(k, n_threads=None, trial_every=3):
    s = [GP.THINK, GP.TEXT, GP.PAR, GP.OUT]
    for i in range(k):
        if i % trial_every == 0:
            s += [GP.TRI, GP.TEXT, GP.END_TRI]
        else:
            s += [GP.SUB, GP.TEXT, GP.TEXT, GP.END_SUB]
    s += [GP.END_OUT]
    for i in range(k if n_threads is None else n_threads):
        s += [GP.THR] + [GP.TEXT] * (i % 5) + [GP.END_THR]
    return s + [GP.END_PAR, GP.END_THINK]


def adversarial_streams():
    rng = np.random.default_rng(11)
    streams = []
    # every valid string up to length 14 plus mutations/truncations of some
    valid = [list(s) for s in GP.enumerate_valid(16)]
    streams += valid[::3]
    for s in valid[::7]:
        i = int(rng.integers(0, len(s)))
        streams.append(s[:i] + [int(rng.integers(0, 13))] + s[i + 1:])
        streams.append(s[: int(rng.integers(0, len(s) + 1))])
    # empty rows, single tokens
    streams += [[], [GP.THINK], [GP.TEXT], [GP.END_THINK]]
    # nesting across the three tiers: LDS frames for 5 levels (rows_fast), for
    # 33 (rows_mid), then global frames (rows_deep)
    streams += [deep_stream(d) for d in (1, 2, 4, 5, 6, 9, 10, 32, 33, 34, 40, 1000)]
    streams.append(deep_stream(300, GP.TRI)[:-5])  # truncated deep
    # fan-out beyond the 64 entries of the fast path, with a thread-count mismatch
    streams += [fanout_stream(64), fanout_stream(65), fanout_stream(200, 150), fanout_stream(70, 90)]
    # dense: tags everywhere (segments overflow their event capacity)
    dense = [GP.THINK]
    for _ in range(2500):
        dense += [GP.PAR, GP.OUT, GP.TRI, GP.TEXT, GP.END_TRI, GP.END_OUT, GP.THR, GP.END_THR, GP.THR, GP.TEXT,
                  GP.END_THR, GP.END_PAR]
    streams.append(dense + [GP.END_THINK, GP.TEXT])
    streams.append(dense[:-3] + [GP.END_THINK])  # invalid deep inside a dense row
    # long text with tags straddling segment boundaries
    long = [GP.THINK] + [GP.TEXT] * 4094 + [GP.PAR, GP.OUT, GP.SUB, GP.TEXT, GP.END_SUB, GP.SUB, GP.TEXT, GP.END_SUB,
                                           GP.END_OUT, GP.THR] + [GP.TEXT] * 9000 + [GP.END_THR, GP.THR, GP.END_THR,
                                                                                      GP.END_PAR, GP.END_THINK]
    streams.append(long)
    streams.append(long[:4097] + [GP.TEXT] + long[4097:])  # misplaced text
    # the repaired Figure 3
    g = json.load(open(os.path.join(os.path.dirname(__file__), "golden", "fig3_repaired.json")))
    streams.append(GP.parse_names(g["stream"]))
    return streams


