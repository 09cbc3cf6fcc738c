"""Pins of the policy-gradient oracle (GRPO advantage, token-level clipped
surrogate with separate clip ratios 0.2 / 0.28 of Sec. 4) against independent
formulations: numpy z-scores, the textbook min/clip objective written with
np.minimum and np.clip, and central finite differences of that objective."""
import numpy as np

from oracle import pg_oracle as PG

EPS_LO, EPS_HI = 0.2, 0.28


def textbook_loss(logp, logp_old, starts, lengths, adv):
    """-(1/N) sum_t min(rho A, clip(rho, 1-eps_lo, 1+eps_hi) A), all in float64."""
    n_tok = int(np.sum(lengths))
    tot = 0.0
    for i in range(len(starts)):
        s, n = starts[i], lengths[i]
        rho = np.exp(logp[s: s + n] - logp_old[s: s + n])
        tot += np.sum(np.minimum(rho * adv[i], np.clip(rho, 1 - EPS_LO, 1 + EPS_HI) * adv[i]))
    return -tot / n_tok


def batch(seed, n_rows=16, spread=0.2):
    rng = np.random.default_rng(seed)
    lengths = rng.integers(1, 60, n_rows).astype(np.int32)
    starts = np.concatenate([[0], np.cumsum(lengths)[:-1]]).astype(np.int64)
    N = int(lengths.sum())
    old = (-rng.random(N) * 6).astype(np.float32)
    new = (old + rng.uniform(-spread, spread, N)).astype(np.float32)
    reward = rng.choice([-1.0, 1.0, 1.3, 0.7], n_rows).astype(np.float32)
    return old, new, starts, lengths, reward


def test_advantages_are_group_zscores():
    rng = np.random.default_rng(0)
    r = rng.normal(size=64).astype(np.float32)
    r[8:16] = 1.25  # an all-equal group
    a = PG.advantages(r, 8)
    x = r.astype(np.float64).reshape(-1, 8)
    with np.errstate(invalid="ignore"):
        ref = (x - x.mean(1, keepdims=True)) / x.std(1, keepdims=True)
    ref[1] = 0.0  # sigma = 0
    np.testing.assert_allclose(a.reshape(-1, 8), ref, rtol=1e-13, atol=1e-13)
    assert np.all(a[8:16] == 0)


def test_surrogate_matches_textbook_objective():
    for seed in range(5):
        old, new, starts, lengths, reward = batch(seed)
        adv = PG.advantages(reward, 8).astype(np.float32)
        res = PG.surrogate(new, old, starts, lengths, adv, EPS_LO, EPS_HI)
        ref = textbook_loss(new.astype(np.float64), old.astype(np.float64), starts, lengths, adv.astype(np.float64))
        # both in float64 from the same inputs: summation order only
        assert abs(res["loss"] - ref) <= 1e-13 * max(1.0, abs(ref))
        assert res["tokens"] == lengths.sum()


def test_gradient_matches_finite_differences():
    old, new, starts, lengths, reward = batch(11, n_rows=8, spread=0.4)
    adv = PG.advantages(reward, 8).astype(np.float32)
    res = PG.surrogate(new, old, starts, lengths, adv, EPS_LO, EPS_HI)
    lp = new.astype(np.float64)
    lo = old.astype(np.float64)
    thr_lo, thr_hi = np.log(1 - EPS_LO), np.log(1 + EPS_HI)
    d = lp - old.astype(np.float64)
    h = 1e-6
    checked = 0
    for t in range(0, lp.size, 3):
        if min(abs(d[t] - thr_hi), abs(d[t] - thr_lo)) < 1e-3:
            continue  # the objective has a kink at the clip bound
        e = np.zeros_like(lp)
        e[t] = h
        fd = (textbook_loss(lp + e, lo, starts, lengths, adv.astype(np.float64))
              - textbook_loss(lp - e, lo, starts, lengths, adv.astype(np.float64))) / (2 * h)
        assert abs(res["grad"][t] - fd) <= 1e-6 * max(1e-3, abs(fd)), (t, res["grad"][t], fd)
        checked += 1
    assert checked > 50
    # clipped tokens have zero gradient and were counted
    assert res["clip_high"] + res["clip_low"] == int(np.sum(res["grad"] == 0) - np.sum(np.repeat(adv, lengths) == 0))


def test_closed_forms():
    old, new, starts, lengths, reward = batch(3)
    # rho = 1 everywhere: grad = -A / N, loss = -(sum_i A_i len_i) / N
    adv = PG.advantages(reward, 8).astype(np.float32)
    res = PG.surrogate(old, old, starts, lengths, adv, EPS_LO, EPS_HI)
    N = lengths.sum()
    np.testing.assert_allclose(res["grad"], -np.repeat(adv.astype(np.float64), lengths) / N, rtol=0, atol=1e-15)
    assert abs(res["loss"] + np.sum(adv.astype(np.float64) * lengths) / N) < 1e-12
    # A = 0: nothing moves
    res = PG.surrogate(new, old, starts, lengths, np.zeros(len(starts), np.float32), EPS_LO, EPS_HI)
    assert res["loss"] == 0 and np.all(res["grad"] == 0) and res["clip_high"] == res["clip_low"] == 0


def test_clip_decision_at_the_bounds():
    """Tokens placed just inside and just outside rho = 1 + eps_high and
    rho = 1 - eps_low: the decision follows the clip bounds of the objective,
    and matches the textbook min/clip form token by token."""
    rng = np.random.default_rng(7)
    n = 4000
    old = (-rng.random(n) * 4).astype(np.float32)
    off = rng.choice([np.log(1 + EPS_HI), np.log(1 - EPS_LO)], n) + rng.uniform(-1e-5, 1e-5, n)
    new = (old.astype(np.float64) + off).astype(np.float32)
    d = new.astype(np.float64) - old.astype(np.float64)
    for a in (1.5, -0.75):
        res = PG.surrogate(new, old, np.array([0]), np.array([n]), np.array([a], np.float32), EPS_LO, EPS_HI)
        rho = np.exp(d)
        want = rho > 1 + EPS_HI if a > 0 else rho < 1 - EPS_LO
        assert np.array_equal(res["clipped"], want)
        assert 100 < want.sum() < n - 100  # both sides of the bound are exercised
        # the textbook form picks the clipped term exactly where it is strictly smaller
        terms = np.minimum(rho * a, np.clip(rho, 1 - EPS_LO, 1 + EPS_HI) * a)
        assert np.array_equal(terms < rho * a, want)
