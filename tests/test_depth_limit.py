"""The documented nesting limit, on both sides: a row nested PARASON_MAX_DEPTH
(2^20) deep is evaluated like any other and matches the oracle; a row one level
deeper is refused with PARASON_FLAG_DEPTH_LIMIT (total = its length, every
other integer output 0), and its group's rewards are NaN.  The oracle itself
evaluates both (it has no such limit), so the test also checks that they are
the valid rows of the depth they were built with.

Each deep row is <think>, then 2^20 (or 2^20 + 1) levels of
<Parallel><Outlines><Subtask> t </Subtask></Outlines><Thread> t, closed in
reverse, then </think>: about 10.5 M tokens.  The rows go through the deep tier
(the first block of group_reward runs it), on the CPU SIMT emulation (one
emulated compute unit) and on the GPU."""
import numpy as np
import pytest

import grammar_pins as GP
from adversarial import adversarial_streams, pack
from gpu_util import DEFAULT_COEF, fetch, oracle_expect, to_dev
from paper_2608_24658_amd import parason as PX
from paper_2608_24658_amd.synth import synth as S

TAGS = S.CONTIGUOUS_TAGS
G = 8
D = PX.MAX_DEPTH


def deep_row(depth):
    tid = lambda c: int(TAGS[c - 1])  # noqa: E731
    text = 7
    level = np.array([tid(GP.PAR), tid(GP.OUT), tid(GP.SUB), text, tid(GP.END_SUB), tid(GP.END_OUT), tid(GP.THR),
                      text], np.int32)
    close = np.array([tid(GP.END_THR), tid(GP.END_PAR)], np.int32)
    return np.concatenate([[tid(GP.THINK)], np.tile(level, depth), np.tile(close, depth), [tid(GP.END_THINK)]]
                          ).astype(np.int32)


def batch():
    """Group A: the row nested D deep and 7 short rows; group B: the row
    nested D + 1 deep and 7 short rows."""
    short_t, short_s, short_l = pack(adversarial_streams()[:14], TAGS)
    shorts = [short_t[s: s + n] for s, n in zip(short_s[:14], short_l[:14])]
    rows = [deep_row(D)] + shorts[:7] + [deep_row(D + 1)] + shorts[7:14]
    lengths = np.array([r.size for r in rows], np.int32)
    starts = np.zeros(len(rows), np.int64)
    starts[1:] = np.cumsum(lengths[:-1])
    correct = (np.arange(len(rows)) % 2 == 0).astype(np.uint8)
    return np.concatenate(rows), starts, lengths, correct


def check(got, tokens, starts, lengths, correct):
    rows, R, rs, rt, eta = oracle_expect(tokens, starts, lengths, correct, TAGS, G, DEFAULT_COEF)
    assert rows["max_depth"][0] == D and rows["max_depth"][8] == D + 1
    assert rows["flags"][0] & PX.FLAG_VALID and rows["flags"][8] & PX.FLAG_VALID
    keep = np.arange(16) != 8
    for k in PX.INT_FIELDS:
        assert np.array_equal(got[k][keep], rows[k][keep]), k
    assert np.array_equal(got["flags"][keep], rows["flags"][keep])
    # the row beyond the limit: refused, not evaluated
    assert got["flags"][8] == PX.FLAG_DEPTH_LIMIT
    assert got["total"][8] == lengths[8]
    for k in ("latency", "n_subtask", "n_trial", "n_blocks", "max_depth", "first_error_pos"):
        assert got[k][8] == 0, k
    # group A: the float rounding of the oracle's rewards; group B: NaN
    assert np.array_equal(got["reward"][:8], R[:8].astype(np.float32))
    assert np.all(np.isnan(got["reward"][8:]))


def test_depth_limit_on_the_emulation(tmp_path):
    import test_simt_emulation as T

    if not __import__("os").path.exists(T.CLANG):
        pytest.skip("no host clang++ with the sanitizers")
    tokens, starts, lengths, correct = batch()
    binary = T.build(str(tmp_path / "emu"))
    got, rc = T.run_emu(binary, tokens, starts, lengths, correct, cus=T.FEW, tmp=str(tmp_path))
    assert rc == PX.OK
    check(got, tokens, starts, lengths, correct)


@pytest.mark.gpu
def test_depth_limit_on_the_gpu():
    import torch

    dev = torch.device("cuda:0")
    print("case depth limit: rows nested %d and %d deep" % (D, D + 1), flush=True)
    tokens, starts, lengths, correct = batch()
    px = PX.Parason(TAGS, group_size=G, **DEFAULT_COEF)
    out = px.run(to_dev(tokens, torch.int32, dev), to_dev(starts, torch.int64, dev), to_dev(lengths, torch.int32, dev),
                 to_dev(correct, torch.uint8, dev))
    torch.cuda.synchronize()
    check(fetch(out), tokens, starts, lengths, correct)
