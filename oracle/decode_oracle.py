"""CPU oracle of the grammar-constrained decode step.

TEST INFRASTRUCTURE.  Only the tests may import this module.

During rollouts the tags are kept valid by constrained decoding (Sec. 3.4:
XGrammar enforces valid tags; Sec. 3.1: the grammar keeps rollouts free of
syntax errors).  The set of tokens a constrained decoder may emit after a
prefix is, by definition, the set of tokens that keep the prefix a prefix of
some valid stream of the grammar of Figure 4 (Sec. 3.2).  This oracle computes
exactly that with the parser of ``parason_oracle.c``: class c is allowed after
`prefix` iff the parser reports prefix + [c] as valid or as truncated (it never
fails inside it); the end-of-sequence token is allowed iff the prefix itself is
a complete valid stream.  Text stands for every id that is not a tag and not
the end-of-sequence id.  ``cfg_flags`` selects the language as for the
accounting (CFG_LENIENT_GAPS: Text runs between the structural tags of a
parallel region).
"""
from __future__ import annotations

import numpy as np

from oracle import oracle as O

TEXT = 0


def allowed_classes(prefix_tokens, tag_ids, text_id: int, cfg_flags: int = 0):
    """(set of allowed classes 0..12, eos_allowed) after the token prefix."""
    prefix = list(int(t) for t in prefix_tokens)
    allowed = set()
    for c in range(13):
        tok = text_id if c == TEXT else int(tag_ids[c - 1])
        r = O.eval_stream(prefix + [tok], tag_ids, cfg_flags)
        if r["flags"] & (O.F_VALID | O.F_TRUNCATED):
            allowed.add(c)
    r = O.eval_stream(prefix, tag_ids, cfg_flags)
    return allowed, bool(r["flags"] & O.F_VALID)


def allowed_batch(prefixes, tag_ids, text_id: int, cfg_flags: int = 0):
    """allowed_classes for many prefixes with one call of the parser: for each
    prefix p the rows p, p + [Text], p + [tag 1], ..., p + [tag 12]."""
    cands = [int(text_id)] + [int(t) for t in tag_ids]
    chunks, starts, lengths = [], [], []
    pos = 0
    for p in prefixes:
        p = [int(t) for t in p]
        for tail in [[]] + [[c] for c in cands]:
            row = p + tail
            chunks.append(row)
            starts.append(pos)
            lengths.append(len(row))
            pos += len(row)
    tokens = np.array([t for c in chunks for t in c] or [0], dtype=np.int32)
    res = O.eval_rows(tokens, np.array(starts, dtype=np.int64), np.array(lengths, dtype=np.int32), tag_ids,
                      cfg_flags)
    out = []
    for i in range(len(prefixes)):
        r = res[14 * i: 14 * (i + 1)]
        allowed = {c for c in range(13) if r[1 + c]["flags"] & (O.F_VALID | O.F_TRUNCATED)}
        out.append((allowed, bool(r[0]["flags"] & O.F_VALID)))
    return out


def prefix_is_viable(prefix_tokens, tag_ids, cfg_flags: int = 0) -> bool:
    r = O.eval_stream(list(int(t) for t in prefix_tokens), tag_ids, cfg_flags)
    return bool(r["flags"] & (O.F_VALID | O.F_TRUNCATED)) or len(prefix_tokens) == 0
