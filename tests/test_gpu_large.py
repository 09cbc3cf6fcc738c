"""The large workload (89,000 groups x 8 rows, mean 50.3k tokens: 3.6e10 tokens,
143 GB of int32) at full size, in the launch configuration the benchmark times.

The oracle cannot take the whole batch in seconds, so: every row's length and
start are recomputed on the host by the generator mirror; a seeded sample of
rows (plus the first and last rows) is regenerated token by token on the host,
checked against the device copy, and evaluated by the oracle; the sampled
groups' rewards are compared too.  Properties that hold at any size are
checked on every row."""
import numpy as np
import pytest

from gpu_util import DEFAULT_COEF, compare, fetch, log
from oracle import oracle as O
from paper_2608_24658_amd import parason as PX
from paper_2608_24658_amd.synth import synth as S

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

G = S.GROUP_SIZE


def test_large_workload_sampled(request):
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    dev = torch.device("cuda:0")
    P = S.make_params("large")
    n = S.n_rows_of("large")
    log("case large: host lengths")
    ln_h, co_h = S.host_rows(P, n)
    st_h = np.zeros(n, np.int64)
    st_h[1:] = np.cumsum(ln_h[:-1].astype(np.int64))
    total = int(ln_h.astype(np.int64).sum())
    log("case large: device generation of %d rows, %d tokens" % (n, total))
    tok_d, st_d, ln_d, co_d = S.device_batch(P, n, device=dev)
    assert np.array_equal(st_d.cpu().numpy(), st_h) and np.array_equal(ln_d.cpu().numpy(), ln_h)
    assert np.array_equal(co_d.cpu().numpy(), co_h)
    px = PX.Parason(S.CONTIGUOUS_TAGS, group_size=G, **DEFAULT_COEF)
    log("case large: run")
    out = px.run(tok_d, st_d, ln_d, co_d, total_tokens=total)
    torch.cuda.synchronize()
    got = fetch(out)

    # properties on every row
    assert np.array_equal(got["total"], ln_h)
    assert np.all(got["latency"] <= got["total"]) and np.all(got["latency"] > 0)
    assert np.all(got["n_subtask"] + got["n_trial"] <= got["total"] - 2)
    assert np.all(got["flags"] & PX.FLAG_VALID)  # every generated large row is complete
    assert np.all(np.isfinite(got["reward"]))
    assert np.all((got["reward"] == -1.0) == ((co_h == 0)))

    # sampled groups, compared in full with the oracle
    rng = np.random.default_rng(3)
    groups = np.unique(np.r_[0, n // G - 1, rng.choice(n // G, 30, replace=False)])
    rows_idx = (groups[:, None] * G + np.arange(G)[None, :]).ravel()
    toks = []
    for r in rows_idx:
        t = S.host_row_tokens(P, int(r), int(st_h[r]), int(ln_h[r]))
        d = tok_d[int(st_h[r]): int(st_h[r]) + int(ln_h[r])].cpu().numpy()
        assert np.array_equal(t, d), "row %d differs from the host mirror" % r
        toks.append(t)
    lens = ln_h[rows_idx]
    starts = np.zeros(rows_idx.size, np.int64)
    starts[1:] = np.cumsum(lens[:-1].astype(np.int64))
    rows = O.eval_rows(np.concatenate(toks), starts, lens, S.CONTIGUOUS_TAGS)
    c = DEFAULT_COEF
    R, rs, rt, eta = O.group_reward(rows, co_h[rows_idx], G, c["alpha"], c["beta_subtask"], c["beta_trial"],
                                    c["rho"], c["rho_clip"])
    n_exact = compare(got, rows, R, rs, rt, eta, idx=rows_idx, what="large sample")
    log("large: %d rows, %d tokens; %d sampled rows match, %d of their rewards bit-exact" % (
        n, total, rows_idx.size, n_exact))
    del tok_d, out
    torch.cuda.empty_cache()
