"""Cases shared by the fork/join tests on the GPU and on the CPU emulation:
synthetic rollouts cut right after one of their </Outlines> tags, hand-made
rows (well formed, rejected, with outlines across 256-token chunk edges, long
outlines), short rows in large numbers, the oracle's expected outputs, buffer
layouts with gaps, and worker sequences handed back to the join."""
import numpy as np

from oracle import fork_oracle as F
from paper_2608_24658_amd.synth import synth as S
from tests import grammar_pins as GP

CONTIG = [int(t) for t in S.CONTIGUOUS_TAGS]
SCATTERED = [91, 5, 40000, 17, 151000, 12, 333, 77777, 2, 64, 99999, 150001]


def synthetic_main_rows(workload, n, tags, seed, p_raw=0.05):
    """Rows of a synthetic workload cut right after a random </Outlines>."""
    P = S.make_params(workload, tag_ids=tags)
    tok, st, ln, _ = S.host_batch(P, n)
    end_out = tags[GP.END_OUT - 1]
    rng = np.random.default_rng(seed)
    rows = []
    for i in range(n):
        row = tok[st[i]: st[i] + ln[i]]
        ends = np.nonzero(row == end_out)[0]
        if len(ends) == 0 or rng.random() < p_raw:
            rows.append(row[: rng.integers(0, len(row) + 1)].tolist())
        else:
            rows.append(row[: int(rng.choice(ends)) + 1].tolist())
    return rows


def hand_rows(tags, text_ids):
    def t(names):
        out = []
        for k, c in enumerate(GP.parse_names(names)):
            out.append(tags[c - 1] if c else text_ids[k % len(text_ids)])
        return out

    rows = [t(x) for x in (
        "think t5 Par Out Sub t3 /Sub Sub t2 /Sub Sub t4 /Sub /Out",
        "think Par Out Sub t /Sub",
        "think t /Out",
        "think Out Sub t /Sub /Out",
        "think Par t Out Sub t /Sub /Out",
        "think Par Out /Out",
        "think Par Out Sub /Sub /Out",
        "think Par Out Sub t /Tri /Out",
        "think Par Out Sub t /Sub t Tri t /Tri /Out",
        "think Par Out t Sub t /Sub /Out",
        "think Par Out Sub t Thr /Sub /Out",
        "/Out",
        "Out /Out",
        "Par Out Tri t /Tri /Out",
        "think Par Out Sub t /Sub /Out Thr t /Thr /Par Par Out Tri t2 /Tri Tri t /Tri /Out",
    )]
    rows += [[], [tags[GP.END_OUT - 1]]]
    # outlines spanning many 256-token chunks: long entry texts, many short entries
    rows.append(t("think t300 Par Out Sub t700 /Sub Tri t1 /Tri Sub t257 /Sub /Out"))
    rows.append(t("think t3 Par Out " + "Sub t /Sub Tri t /Tri " * 300 + "/Out"))
    rows.append(t("think t3 Par Out " + "Sub t /Sub Tri t /Tri " * 300 + "Sub /Sub /Out"))  # last entry empty
    rows.append(t("think t900 Par t2 Out " + "Tri t40 /Tri " * 30 + "/Out"))  # <Parallel> text <Outlines>
    # the <Outlines> sits exactly on chunk edges
    for pad in (250, 251, 252, 253, 254, 255, 256, 257):
        rows.append(t("think t%d Par Out Sub t2 /Sub /Out" % pad))
    return rows


def oracle_fork(rows, tags, seed, lenient=False):
    res = F.fork(rows, tags, flags=F.FORK_SEED_ENTRY if seed else 0, lenient=lenient)
    lens = np.array([len(c) for c in res["ctx"]], dtype=np.int64)
    starts = np.zeros(len(lens), dtype=np.int64)
    if len(lens):
        starts[1:] = np.cumsum(lens[:-1])
    flat = np.array([x for c in res["ctx"] for x in c], dtype=np.int32)
    return res, starts, lens, flat


def layout(rows, rng, gaps=True, shuffle=True):
    """Rows placed in one buffer in a random order with random gaps."""
    order = rng.permutation(len(rows)) if shuffle else np.arange(len(rows))
    starts = np.zeros(len(rows), dtype=np.int64)
    pieces = []
    pos = 0
    for i in order:
        g = int(rng.integers(0, 5)) if gaps else 0
        pieces.append(np.zeros(g, np.int32))
        pos += g
        starts[i] = pos
        pieces.append(np.asarray(rows[i], dtype=np.int32))
        pos += len(rows[i])
    buf = np.concatenate(pieces) if pieces else np.zeros(0, np.int32)
    return (buf if buf.size else np.zeros(1, np.int32)), starts, np.array([len(r) for r in rows], dtype=np.int32)


def worker_sequences(res, tags, rng, p_bad=0.0):
    thr_end = tags[GP.END_THR - 1]
    seqs = []
    for c in res["ctx"]:
        gen = [int(x) for x in rng.integers(0, 1000, size=int(rng.integers(0, 60)))]
        s = list(c) + gen + [thr_end]
        if rng.random() < p_bad:
            s = s[: int(rng.integers(0, len(s)))]  # cut anywhere, even inside the row
        seqs.append(s)
    return seqs


def short_rows(tags, n, rng):
    """n short rows: well-formed outlines of 1..4 entries, malformed ones and
    empty rows, so that many rows give few tokens."""
    base = hand_rows(tags, [7, 8, 9, 1000, 150000])[:17]
    rows = []
    for i in range(n):
        k = int(rng.integers(0, 6))
        if k < 4:
            names = "think t%d Par Out " % int(rng.integers(1, 9)) + " ".join(
                ("Sub t%d /Sub" if rng.random() < 0.5 else "Tri t%d /Tri") % int(rng.integers(1, 5))
                for _ in range(k + 1)) + " /Out"
            rows.append([tags[c - 1] if c else 7 for c in GP.parse_names(names)])
        else:
            rows.append(list(base[int(rng.integers(0, len(base)))]))
    return rows


def lenient_hand_rows(tags, text_ids):
    def t(names):
        out = []
        for k, c in enumerate(GP.parse_names(names)):
            out.append(tags[c - 1] if c else text_ids[k % len(text_ids)])
        return out

    rows = [t(x) for x in (
        "think Par t Out t Sub t3 /Sub t2 Tri t /Tri t /Out",
        "think Par t2 Out Sub t /Sub /Out",
        "think Par Out t Sub t /Sub t Tri t2 /Tri /Out",
        "think Par Out t /Out",
        "think Par t t Out",
        "think Thr t Out Sub t /Sub /Out",
        "think Par Out Sub t /Sub t /Out Thr t /Thr t /Par Par t Out t Tri t2 /Tri t Tri t /Tri t3 /Out",
        "think Par Out Sub /Sub t /Out",
    )]
    # a gap before <Outlines> that spans chunks, and gaps between many entries
    rows.append(t("think t5 Par t600 Out Sub t2 /Sub /Out"))
    rows.append(t("think Par t300 Out t300 " + "Sub t /Sub t3 Tri t2 /Tri " * 200 + "t500 /Out"))
    for pad in (250, 253, 254, 255, 256):  # <Outlines> and the first entry near chunk edges
        rows.append(t("think Par t%d Out t%d Sub t2 /Sub t /Out" % (pad, 256 - pad % 7)))
    return rows
