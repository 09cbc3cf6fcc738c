"""GPU parity of the policy-gradient step (advantages, clipped surrogate and
its gradient) against the CPU oracle on the same seeded inputs.

The oracle decides clipping by its definition, rho = exp(logp - logp_old) in
float64 against 1 + eps_high and 1 - eps_low.  The kernel decides on the float
log-ratio d = logp - logp_old against float ln(1 + eps_high), ln(1 - eps_low).
Rounding is monotone, so the two can differ only for a token whose float64 d
rounds to the same float as a threshold (within one float rounding of
ln(1 +- eps)): such boundary tokens are counted, logged and bounded, and there
the kernel may take either decision.  Every other token's decision must be
the oracle's.

Tolerances: the kernel's clip counts equal its own per-token decisions (read
from its gradient: zero exactly where it clipped) and the token count is exact.
Advantages: the kernel evaluates the same double expression in the same order
and stores float, so within 2^-24 |A|.  Gradient: the kernel takes
rho = expf(d) and -(A * rho) * (1/N) in float (a few float roundings) against
the oracle's double values: 2^-20 relative, plus 1e-30 absolute.  Loss: float
terms summed in double: 2^-20 relative, plus, per boundary token, the gap
between its two terms (at most 2^-20 |A| / N)."""
import numpy as np
import pytest

from gpu_util import log, to_dev
from oracle import oracle as O
from oracle import pg_oracle as PG
from paper_2608_24658_amd import parason as PX
from paper_2608_24658_amd.synth import synth as S

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

G = S.GROUP_SIZE
EPS_LO, EPS_HI = 0.2, 0.28
TOL = 2.0 ** -20


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch.device("cuda:0")


def rewards_for(P, n):
    tok, st, ln, co = S.host_batch(P, n)
    rows = O.eval_rows(tok, st, ln, S.CONTIGUOUS_TAGS)
    R, *_ = O.group_reward(rows, co, G, 0.1, 0.0, 0.1, 0.5, 0.25)
    return R.astype(np.float32), st, ln


def boundary_tokens(d):
    """Tokens whose float64 log-ratio d rounds to the same float as one of the
    kernel's float thresholds: the only ones the two decisions may differ on."""
    thr_lo, thr_hi = np.float32(np.log1p(-EPS_LO)), np.float32(np.log1p(EPS_HI))
    d32 = d.astype(np.float32)
    return (d32 == thr_lo) | (d32 == thr_hi)


def check_rows(g, exp, adv_row, lengths, what):
    """Per-token comparison of the gradient g (float64, the oracle's layout)
    with the oracle; returns the kernel's per-token clip decisions and the
    number of boundary tokens."""
    inside = ~np.isnan(exp["grad"])
    a = np.repeat(np.asarray(adv_row, np.float32).astype(np.float64), np.maximum(lengths, 0))
    gi, ei, di = g[inside], exp["grad"][inside], exp["d"][inside]
    bnd = boundary_tokens(di)
    gpu_clipped = (gi == 0) & (a != 0)
    ora_clipped = exp["clipped"][inside]
    bad = (gpu_clipped != ora_clipped) & ~bnd
    assert not np.any(bad), (what, "clip decisions differ off the boundary", int(bad.sum()))
    err = np.abs(gi - ei)
    lim = TOL * np.abs(ei) + 1e-30
    same = gpu_clipped == ora_clipped
    assert np.all(err[same] <= lim[same]), (what, float(np.max(err[same] / np.maximum(lim[same], 1e-300))))
    # a boundary token the kernel did not clip carries the unclipped gradient
    unc = ~gpu_clipped & ~same
    if np.any(unc):
        n_tok = exp["tokens"]
        want = -a[unc] * np.exp(di[unc]) / n_tok
        assert np.all(np.abs(gi[unc] - want) <= TOL * np.abs(want) + 1e-30), what
    n_bnd = int(bnd.sum())
    assert n_bnd <= max(8, 1e-6 * inside.sum()), (what, n_bnd)
    return gpu_clipped, a, n_bnd


def check(got, exp, adv_exp, starts, lengths, what):
    adv = got["advantage"].cpu().numpy().astype(np.float64)
    assert np.all(np.abs(adv - adv_exp) <= 2.0 ** -24 * np.abs(adv_exp)), what
    g = got["grad"].cpu().numpy().astype(np.float64)
    inside = ~np.isnan(exp["grad"])
    gpu_clipped, a, n_bnd = check_rows(g, exp, adv_exp.astype(np.float32), lengths, what)
    st = got["stats"].cpu().numpy()
    assert st[1] == exp["tokens"], (what, st, exp["tokens"])
    assert st[2] == int(np.sum(gpu_clipped & (a > 0))) and st[3] == int(np.sum(gpu_clipped & (a < 0))), (what, st)
    slack = n_bnd * 2.0 ** -20 * float(np.max(np.abs(adv_exp), initial=0.0)) / max(1, exp["tokens"])
    assert abs(st[0] - exp["loss"]) <= TOL * max(1e-6, abs(exp["loss"])) + slack, (what, st[0], exp["loss"])
    log("%s: %d boundary tokens; clipped high %d (oracle %d), low %d (oracle %d)" % (
        what, n_bnd, int(st[2]), exp["clip_high"], int(st[3]), exp["clip_low"]))
    return g, inside


@pytest.mark.parametrize("workload", ["tiny", "small", "ragged", "typical"])
def test_pg_parity(dev, workload):
    log("case pg %s" % workload)
    P = S.make_params(workload)
    n = S.n_rows_of(workload)
    reward, starts, lengths = rewards_for(P, n)
    N = int(lengths.astype(np.int64).sum())
    old_d, new_d = S.device_logp(P, N, device=dev)
    old_h, new_h = S.host_logp(P, 0, N)
    assert np.array_equal(old_d.cpu().numpy(), old_h) and np.array_equal(new_d.cpu().numpy(), new_h)
    got = PX.pg_run(to_dev(reward, torch.float32, dev), new_d, old_d, to_dev(starts, torch.int64, dev),
                    to_dev(lengths, torch.int32, dev), G, EPS_LO, EPS_HI)
    torch.cuda.synchronize()
    adv_exp = PG.advantages(reward, G)
    exp = PG.surrogate(new_h, old_h, starts, lengths, adv_exp.astype(np.float32), EPS_LO, EPS_HI)
    check(got, exp, adv_exp, starts, lengths, workload)
    log("%s: %d tokens, loss %.6g, clipped %d/%d" % (workload, N, exp["loss"], exp["clip_high"], exp["clip_low"]))


def test_pg_layout_gaps_and_misalignment(dev):
    """Padded rows at every alignment: positions outside rows are not written."""
    log("case pg layout")
    rng = np.random.default_rng(5)
    n = 24
    lengths = rng.integers(0, 3000, n).astype(np.int32)
    lengths[3] = 1
    lmax = int(lengths.max()) + 5
    starts = (np.arange(n) * lmax + 1).astype(np.int64)
    total = n * lmax + 8
    P = S.make_params("small")
    old_h, new_h = S.host_logp(P, 0, total)
    reward = rng.choice([-1.0, 0.5, 1.0, 1.7], n).astype(np.float32)
    reward[16:24] = 1.0  # an all-equal group: A = 0
    for shift in (0, 1, 3):
        buf_o = to_dev(np.concatenate([np.zeros(shift, np.float32), old_h]), torch.float32, dev)[shift:]
        buf_n = to_dev(np.concatenate([np.zeros(shift, np.float32), new_h]), torch.float32, dev)[shift:]
        grad = to_dev(np.concatenate([np.zeros(shift, np.float32), np.full(total, 7.5, np.float32)]),
                      torch.float32, dev)[shift:]
        got = PX.pg_run(to_dev(reward, torch.float32, dev), buf_n, buf_o, to_dev(starts, torch.int64, dev),
                        to_dev(lengths, torch.int32, dev), G, EPS_LO, EPS_HI, grad=grad)
        torch.cuda.synchronize()
        adv_exp = PG.advantages(reward, G)
        exp = PG.surrogate(new_h, old_h, starts, lengths, adv_exp.astype(np.float32), EPS_LO, EPS_HI)
        g, inside = check(got, exp, adv_exp, starts, lengths, "shift %d" % shift)
        assert np.all(g[~inside] == 7.5)


def test_pg_rows_without_tokens(dev):
    """Rows that are all empty: there is no token, so the loss, the token count
    and the clip counts are 0, the advantages are still each group's, and the
    gradient buffer is left as it was."""
    log("case pg rows without tokens")
    n = 16
    starts = np.zeros(n, np.int64)
    lengths = np.zeros(n, np.int32)
    reward = np.random.default_rng(9).choice([-1.0, 0.5, 1.0], n).astype(np.float32)
    logp = np.zeros(4, np.float32)
    grad = to_dev(np.full(4, 7.5, np.float32), torch.float32, dev)
    got = PX.pg_run(to_dev(reward, torch.float32, dev), to_dev(logp, torch.float32, dev),
                    to_dev(logp, torch.float32, dev), to_dev(starts, torch.int64, dev),
                    to_dev(lengths, torch.int32, dev), G, EPS_LO, EPS_HI, grad=grad)
    torch.cuda.synchronize()
    adv_exp = PG.advantages(reward, G)
    exp = PG.surrogate(logp, logp, starts, lengths, adv_exp.astype(np.float32), EPS_LO, EPS_HI)
    assert exp["tokens"] == 0 and exp["loss"] == 0.0
    check(got, exp, adv_exp, starts, lengths, "no tokens")
    assert np.all(got["grad"].cpu().numpy() == 7.5)
    assert np.all(got["stats"].cpu().numpy() == 0.0)


def test_pg_wide_log_ratio(dev):
    """Log-ratios over [-70, 88]: rows of positive advantage keep the tokens
    with d <= ln 1.28 (ratios down to 4e-31), rows of negative advantage those
    with d >= ln 0.8 (ratios up to 1.6e38), so the kept gradients check the
    kernel's exponential against the oracle's exp in double at the 2^-20 bound
    over the range where the gradient -A rho / N stays a normal float (below
    it a kept token's gradient could underflow to the zero that marks a
    clipped one)."""
    log("case pg wide log-ratio")
    rng = np.random.default_rng(11)
    n, row_len = 64, 16384
    d = rng.permutation(np.linspace(-70.0, 88.0, n * row_len).astype(np.float32))
    old_h = np.where(np.arange(d.size) % 2 == 0, np.float32(0.0), np.float32(-3.0)).astype(np.float32)
    new_h = (old_h + d).astype(np.float32)
    starts = (np.arange(n) * row_len).astype(np.int64)
    lengths = np.full(n, row_len, np.int32)
    reward = np.tile(np.array([1.0, 0.0], np.float32), n // 2)  # A = +1, -1 alternately
    got = PX.pg_run(to_dev(reward, torch.float32, dev), to_dev(new_h, torch.float32, dev),
                    to_dev(old_h, torch.float32, dev), to_dev(starts, torch.int64, dev),
                    to_dev(lengths, torch.int32, dev), G, EPS_LO, EPS_HI)
    torch.cuda.synchronize()
    adv_exp = PG.advantages(reward, G)
    assert set(np.unique(adv_exp).tolist()) == {-1.0, 1.0}
    exp = PG.surrogate(new_h, old_h, starts, lengths, adv_exp.astype(np.float32), EPS_LO, EPS_HI)
    g, _ = check(got, exp, adv_exp, starts, lengths, "wide log-ratio")
    kept = g != 0
    assert np.any(kept & (exp["d"] < -65)) and np.any(kept & (exp["d"] > 80))


def test_pg_rejects_bad_arguments(dev):
    log("case pg args")
    t = torch.zeros(64, dtype=torch.float32, device=dev)
    st = torch.zeros(8, dtype=torch.int64, device=dev)
    ln = torch.zeros(8, dtype=torch.int32, device=dev)
    with pytest.raises(PX.ParasonError):
        PX.pg_run(t[:8], t, t, st, ln, group_size=3)  # 8 rows, G = 3
    with pytest.raises(PX.ParasonError):
        PX.pg_run(t[:8], t, t, st, ln, clip_low=1.0)
    with pytest.raises(PX.ParasonError):
        PX.pg_run(t[:8], t[1:33], t[:32], st, ln)  # different alignment modulo 16 bytes


def test_pg_large_half_sampled(dev):
    """The configuration bench.py --step pg times: the first 356,000 rows of the
    large workload (1.79e10 tokens, logp + logp_old + grad = 215 GB).  The
    gradient of 48 sampled rows (every position, so every clip decision) and
    the advantages of all groups are compared with the oracle; the token count
    is exact."""
    log("case pg large half (215 GB)")
    P = S.make_params("large")
    n = S.n_rows_of("large") // 2 // G * G
    lengths, _ = S.host_rows(P, n)
    starts = np.zeros(n, np.int64)
    starts[1:] = np.cumsum(lengths[:-1].astype(np.int64))
    N = int(lengths.astype(np.int64).sum())
    rng = np.random.default_rng(5)
    reward = rng.choice([-1.0, 1.0, 1.25, 0.8, 1.5], n).astype(np.float32)
    old_d, new_d = S.device_logp(P, N, device=dev)
    grad = torch.empty_like(new_d)
    got = PX.pg_run(to_dev(reward, torch.float32, dev), new_d, old_d, to_dev(starts, torch.int64, dev),
                    to_dev(lengths, torch.int32, dev), G, EPS_LO, EPS_HI, grad=grad)
    torch.cuda.synchronize()
    adv_exp = PG.advantages(reward, G)
    adv = got["advantage"].cpu().numpy().astype(np.float64)
    assert np.all(np.abs(adv - adv_exp) <= 2.0 ** -24 * np.abs(adv_exp))
    st = got["stats"].cpu().numpy()
    assert st[1] == N and 0 <= st[2] + st[3] <= N and np.isfinite(st[0])
    for i in sorted(rng.choice(n, size=48, replace=False).tolist()):
        s0, ln = int(starts[i]), int(lengths[i])
        old_h, new_h = S.host_logp(P, s0, ln)
        exp = PG.surrogate(new_h, old_h, np.array([0]), np.array([ln]), adv_exp[i: i + 1].astype(np.float32),
                           EPS_LO, EPS_HI, n_tokens=N)
        g = grad[s0: s0 + ln].cpu().numpy().astype(np.float64)
        check_rows(g, exp, adv_exp[i: i + 1].astype(np.float32), np.array([ln]), "large half row %d" % i)
    del old_d, new_d, grad
    torch.cuda.empty_cache()
