"""GPU parity of the batch metrics (Tables 2, 4 and 5 definitions) and of the
batch-wide normalisation mode, against the CPU oracle.

Tolerances: counts and token sums are exact; ratios and means of token counts
are one double division of exact integers on both sides, so they must agree
to 1e-15 relative.  The mean reward is taken over the stored float rewards on
the GPU and over the oracle's double rewards, so it agrees to the float reward
bound (2^-23 relative).  Batch-wide mu and sigma are summed in a different
(fixed) order on the GPU than in the oracle's sequential loop; the resulting
rewards are checked with the usual float bound."""
import numpy as np
import pytest

from gpu_util import DEFAULT_COEF, compare, fetch, log, oracle_expect, run_gpu, to_dev
from oracle import oracle as O
from paper_2608_24658_amd import parason as PX
from paper_2608_24658_amd.synth import synth as S

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

G = S.GROUP_SIZE
TAGS = S.CONTIGUOUS_TAGS
EXACT = ("rows", "valid", "triggered", "correct", "truncated", "count_mismatch", "sum_total", "sum_latency",
         "sum_subtask", "sum_trial")


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch.device("cuda:0")


def check_metrics(got_m, rows, correct, R):
    exp = O.batch_metrics(rows, correct, R)
    for i, name in enumerate(PX.METRICS):
        g, e = float(got_m[i]), exp[name]
        if name in EXACT:
            assert g == e, (name, g, e)
        elif name == "mean_reward":
            assert abs(g - e) <= 2.0 ** -23 * max(1.0, np.mean(np.maximum(1.0, np.abs(R)))), (name, g, e)
        else:
            assert abs(g - e) <= 1e-15 * max(1.0, abs(e)), (name, g, e)
    return exp


@pytest.mark.parametrize("workload", ["small", "ragged", "typical"])
def test_metrics_parity(dev, workload):
    log("case metrics %s" % workload)
    P = S.make_params(workload)
    n = S.n_rows_of(workload)
    tok_h, st_h, ln_h, co_h = S.host_batch(P, n)
    px = PX.Parason(TAGS, group_size=G, **DEFAULT_COEF)
    out = px.run(to_dev(tok_h, torch.int32, dev), to_dev(st_h, torch.int64, dev), to_dev(ln_h, torch.int32, dev),
                 to_dev(co_h, torch.uint8, dev), metrics=True)
    torch.cuda.synchronize()
    got = fetch(out)
    rows, R, rs, rt, eta = oracle_expect(tok_h, st_h, ln_h, co_h, TAGS, G, DEFAULT_COEF)
    compare(got, rows, R, rs, rt, eta, what=workload)
    exp = check_metrics(got["metrics"], rows, co_h, R)
    log("%s: trigger %.3f acceleration %.3f mean latency %.0f" % (
        workload, exp["trigger_ratio"], exp["acceleration"], exp["mean_latency"]))


@pytest.mark.parametrize("workload", ["tiny", "small", "ragged", "typical"])
def test_batch_stats_parity(dev, workload):
    log("case batch stats %s" % workload)
    P = S.make_params(workload)
    n = S.n_rows_of(workload)
    tok_h, st_h, ln_h, co_h = S.host_batch(P, n)
    coef = dict(alpha=0.1, beta_subtask=0.05, beta_trial=0.1, rho=0.5, rho_clip=0.25)
    px = PX.Parason(TAGS, group_size=G, flags=PX.CFG_BATCH_STATS, **coef)
    out = px.run(to_dev(tok_h, torch.int32, dev), to_dev(st_h, torch.int64, dev), to_dev(ln_h, torch.int32, dev),
                 to_dev(co_h, torch.uint8, dev), metrics=True)
    torch.cuda.synchronize()
    got = fetch(out)
    rows, R, rs, rt, eta = oracle_expect(tok_h, st_h, ln_h, co_h, TAGS, G, coef, O.CFG_BATCH_STATS)
    compare(got, rows, R, rs, rt, eta, what="batch " + workload, exact_reward=False)
    check_metrics(got["metrics"], rows, co_h, R)


def test_batch_stats_constant_batch_and_not_evaluated(dev):
    log("case batch stats edge")
    # every row identical: sigma = 0 exactly, z = 0
    one = np.array([TAGS[0]] + [5] * 40 + [TAGS[1]], np.int32)
    n = 16
    toks = np.tile(one, n)
    lens = np.full(n, one.size, np.int32)
    starts = (np.arange(n) * one.size).astype(np.int64)
    co = np.ones(n, np.uint8)
    px = PX.Parason(TAGS, group_size=G, flags=PX.CFG_BATCH_STATS, **DEFAULT_COEF)
    got = run_gpu(px, to_dev(toks, torch.int32, dev), to_dev(starts, torch.int64, dev), to_dev(lens, torch.int32, dev),
                  to_dev(co, torch.uint8, dev))
    assert np.all(got["reward"] == 1.0)  # 1 + 2 min(rho * 0, clip)
    # a row that is not evaluated makes the whole batch NaN
    lens_bad = lens.copy()
    lens_bad[3] = -1
    got = run_gpu(px, to_dev(toks, torch.int32, dev), to_dev(starts, torch.int64, dev),
                  to_dev(lens_bad, torch.int32, dev), to_dev(co, torch.uint8, dev))
    assert got["flags"][3] == PX.FLAG_BAD_ROW and np.all(np.isnan(got["reward"]))


def test_metrics_on_large_workload_properties(dev):
    """Properties of the 143 GB workload's metrics that hold at any size: the
    reduction agrees with numpy sums over the fetched per-row outputs (no
    oracle involved: the per-row values are checked against the oracle on
    sampled rows in test_gpu_large), every row counts, and the token total is
    the generator's."""
    log("case metrics large")
    P = S.make_params("large")
    n = S.n_rows_of("large")
    tok_d, st_d, ln_d, co_d = S.device_batch(P, n, device=dev)
    px = PX.Parason(TAGS, group_size=G, **DEFAULT_COEF)
    out = px.run(tok_d, st_d, ln_d, co_d, metrics=True, total_tokens=int(tok_d.numel()))
    torch.cuda.synchronize()
    got = fetch(out)
    m = dict(zip(PX.METRICS, got["metrics"].tolist()))
    fl = got["flags"]
    valid = (fl & PX.FLAG_VALID) != 0
    correct = co_d.cpu().numpy() != 0
    tot = got["total"].astype(np.int64)
    lat = got["latency"].astype(np.int64)
    assert m["rows"] == n and m["sum_total"] == tok_d.numel() == tot.sum()
    assert m["valid"] == valid.sum() and m["triggered"] == ((fl & PX.FLAG_TRIGGERED) != 0).sum()
    assert m["truncated"] == ((fl & PX.FLAG_TRUNCATED) != 0).sum()
    assert m["count_mismatch"] == ((fl & PX.FLAG_COUNT_MISMATCH) != 0).sum()
    assert m["correct"] == correct.sum() and m["accuracy"] == correct.sum() / n
    assert m["sum_latency"] == lat.sum()
    assert m["sum_subtask"] == got["n_subtask"].astype(np.int64).sum()
    assert m["sum_trial"] == got["n_trial"].astype(np.int64).sum()
    assert abs(m["acceleration"] - tot.sum() / lat.sum()) <= 1e-15 * m["acceleration"]
    assert abs(m["mean_latency"] - lat.sum() / n) <= 1e-15 * m["mean_latency"]
    assert abs(m["mean_reward"] - got["reward"].astype(np.float64).mean()) <= 1e-6
    assert 0 <= m["trigger_ratio"] <= 1 and 0 <= m["accuracy"] <= 1
    del tok_d, out
    torch.cuda.empty_cache()


@pytest.mark.parametrize("n_rows", [64, 12288])
@pytest.mark.parametrize("batch_stats", [False, True])
def test_deep_rows_with_metrics(dev, n_rows, batch_stats):
    """Rows nested beyond the LDS tiers (34-60 deep) mixed with shallow ones,
    under both normalisations and with the batch metrics: the deep tier runs
    inside the per-group reward launch, or as a launch of its own before the
    batch-wide statistics.  64 rows take the one-wave row kernel, 12,288 the
    per-lane one."""
    from adversarial import deep_stream, pack
    import grammar_pins as GP

    log("case deep rows n=%d batch_stats=%s" % (n_rows, batch_stats))
    rng = np.random.default_rng(n_rows + batch_stats)
    depths = np.concatenate([rng.integers(34, 61, size=6), rng.integers(6, 34, size=n_rows // 4),
                             rng.integers(1, 6, size=n_rows - 6 - n_rows // 4)])
    rng.shuffle(depths)
    streams = [deep_stream(int(d), GP.TRI if d % 2 else GP.SUB) for d in depths]
    tokens, starts, lengths = pack(streams, TAGS)
    n = lengths.size
    co = (np.arange(n) % 4 != 0).astype(np.uint8)
    flags = PX.CFG_BATCH_STATS if batch_stats else 0
    px = PX.Parason(TAGS, group_size=G, flags=flags, **DEFAULT_COEF)
    out = px.run(to_dev(tokens, torch.int32, dev), to_dev(starts, torch.int64, dev), to_dev(lengths, torch.int32, dev),
                 to_dev(co, torch.uint8, dev), metrics=True)
    torch.cuda.synchronize()
    got = fetch(out)
    rows, R, rs, rt, eta = oracle_expect(tokens, starts, lengths, co, TAGS, G, DEFAULT_COEF,
                                         O.CFG_BATCH_STATS if batch_stats else 0)
    compare(got, rows, R, rs, rt, eta, what="deep rows", exact_reward=not batch_stats)
    check_metrics(got["metrics"], rows, co, R)
    assert int(np.max(got["max_depth"])) >= 34
