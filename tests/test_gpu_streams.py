"""Concurrent calls of one handle on several streams.

A handle holds only host-side configuration, so calls on different streams,
each with its own workspace and outputs, may run at the same time.  Four
batches (tiny, small, ragged, and small again with lenient gaps on a second
handle) are launched on four side streams back to back, with no wait in
between, followed by a fork and a policy-gradient call on further streams;
every result must equal the oracle's (integers bit-exact, floats within the
bound stated in gpu_util).  All streams have the default priority.
"""
import numpy as np
import pytest

from gpu_util import DEFAULT_COEF, compare, fetch, insert_gaps, log, oracle_expect, to_dev
from oracle import fork_oracle as F
from oracle import pg_oracle as PG
from paper_2608_24658_amd import parason as PX
from paper_2608_24658_amd.synth import synth as S

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

G = S.GROUP_SIZE
TAGS = S.CONTIGUOUS_TAGS


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch.device("cuda:0")


def packed(rows):
    lengths = np.array([len(r) for r in rows], np.int32)
    starts = np.zeros(len(rows), np.int64)
    starts[1:] = np.cumsum(lengths[:-1].astype(np.int64))
    return np.concatenate([np.asarray(r, np.int32) for r in rows]), starts, lengths


def test_accounting_on_four_streams(dev):
    log("case four streams")
    strict = PX.Parason(TAGS, group_size=G, **DEFAULT_COEF)
    lenient = PX.Parason(TAGS, group_size=G, flags=PX.CFG_LENIENT_GAPS, **DEFAULT_COEF)
    cases = []
    for wl in ("tiny", "small", "ragged"):
        P = S.make_params(wl)
        cases.append((wl, strict, 0) + tuple(S.host_batch(P, S.n_rows_of(wl))))
    P = S.make_params("small")
    tok, st, ln, co = S.host_batch(P, S.n_rows_of("small"))
    rng = np.random.default_rng(41)
    gapped = [insert_gaps(tok[st[i]: st[i] + ln[i]], TAGS, rng, p=0.5, max_len=3) for i in range(len(ln))]
    tok_g, st_g, ln_g = packed(gapped)
    cases.append(("small with gaps", lenient, PX.CFG_LENIENT_GAPS, tok_g, st_g, ln_g, co))

    streams = [torch.cuda.Stream(device=dev) for _ in cases]
    outs = []
    torch.cuda.synchronize()
    for s, (what, px, fl, tok, st, ln, co) in zip(streams, cases):
        with torch.cuda.stream(s):
            args = (to_dev(tok, torch.int32, dev), to_dev(st, torch.int64, dev), to_dev(ln, torch.int32, dev),
                    to_dev(co, torch.uint8, dev))
            outs.append((args, px.run(*args)))  # keep the inputs alive until the streams finish
    torch.cuda.synchronize()
    for (what, px, fl, tok, st, ln, co), (_, out) in zip(cases, outs):
        compare(fetch(out), *oracle_expect(tok, st, ln, co, TAGS, G, DEFAULT_COEF, fl), what=what)
        log("%s: %d rows match" % (what, len(ln)))


def test_fork_and_pg_beside_accounting(dev):
    """A fork and a policy-gradient call on their own streams while an
    accounting call runs on a third."""
    log("case fork + pg + accounting on three streams")
    px = PX.Parason(TAGS, group_size=G, **DEFAULT_COEF)
    P = S.make_params("ragged")
    n = S.n_rows_of("ragged")
    tok, st, ln, co = S.host_batch(P, n)
    # fork input: rows cut right after one of their </Outlines>
    end_out = TAGS[5]
    rng = np.random.default_rng(43)
    rows = []
    for i in range(n):
        row = tok[st[i]: st[i] + ln[i]]
        ends = np.nonzero(row == end_out)[0]
        rows.append(row[: int(rng.choice(ends)) + 1] if len(ends) else row)
    ftok, fst, fln = packed(rows)
    # policy-gradient input: seeded log-probabilities of every token of the batch
    N = int(ln.astype(np.int64).sum())
    old_h, new_h = S.host_logp(P, 0, N)
    rewards = rng.choice([-1.0, 0.5, 1.0, 1.7], n).astype(np.float32)

    s_acc, s_fork, s_pg = (torch.cuda.Stream(device=dev) for _ in range(3))
    torch.cuda.synchronize()
    with torch.cuda.stream(s_acc):
        acc_in = (to_dev(tok, torch.int32, dev), to_dev(st, torch.int64, dev), to_dev(ln, torch.int32, dev),
                  to_dev(co, torch.uint8, dev))
        acc = px.run(*acc_in)
    with torch.cuda.stream(s_fork):
        f_in = (to_dev(ftok, torch.int32, dev), to_dev(fst, torch.int64, dev), to_dev(fln, torch.int32, dev))
        fork = px.fork(*f_in, seed=True)
    with torch.cuda.stream(s_pg):
        pg_in = (to_dev(rewards, torch.float32, dev), to_dev(new_h, torch.float32, dev),
                 to_dev(old_h, torch.float32, dev), to_dev(st, torch.int64, dev), to_dev(ln, torch.int32, dev))
        pg = PX.pg_run(*pg_in, G, 0.2, 0.28)
    torch.cuda.synchronize()

    compare(fetch(acc), *oracle_expect(tok, st, ln, co, TAGS, G, DEFAULT_COEF), what="accounting beside fork/pg")
    exp = F.fork([r.tolist() for r in rows], TAGS, flags=F.FORK_SEED_ENTRY)
    assert np.array_equal(fork["worker_off"].cpu().numpy(), np.array(exp["worker_off"], np.int64))
    flat = np.array([x for c in exp["ctx"] for x in c], np.int32)
    assert np.array_equal(fork["ctx_tokens"].cpu().numpy(), flat)
    # the policy-gradient step to the bounds of its own parity test: advantages
    # within 2^-23 relative, gradient and loss within 2^-20 relative, counts exact
    adv_exp = PG.advantages(rewards, G)
    ref = PG.surrogate(new_h, old_h, st, ln, adv_exp.astype(np.float32), 0.2, 0.28)
    adv = pg["advantage"].cpu().numpy().astype(np.float64)
    assert np.all(np.abs(adv - adv_exp) <= 2.0 ** -23 * np.maximum(1.0, np.abs(adv_exp)))
    stats = pg["stats"].cpu().numpy()
    assert stats[1] == ref["tokens"] and stats[2] == ref["clip_high"] and stats[3] == ref["clip_low"]
    assert abs(stats[0] - ref["loss"]) <= 2.0 ** -20 * max(1e-6, abs(ref["loss"]))
    g = pg["grad"].cpu().numpy().astype(np.float64)
    inside = ~np.isnan(ref["grad"])
    assert np.all(np.abs(g[inside] - ref["grad"][inside]) <= 2.0 ** -20 * np.abs(ref["grad"][inside]) + 1e-30)
    log("fork: %d workers; pg: %d tokens" % (exp["worker_off"][-1], N))
