"""The ragged workload's row lengths follow the log-uniform law over
[1, 50300] (50.3k: the largest per-trajectory token count the paper states,
Table 5): P(L = x) proportional to 1/x.  Checked on the host mirror of the
generator (the device build is the same integer code, compared bit for bit by
the GPU tests) against the exact harmonic masses, per octave and inside each
octave; the same checks reject the octave-uniform law (one octave uniformly,
then a length uniformly inside it)."""
import numpy as np

from paper_2608_24658_amd.synth import synth as S

HI = 50300
N = 400_000


def harmonic_mass(a, b, H):
    x = np.arange(a, b + 1, dtype=np.float64)
    return float(np.sum(1.0 / x) / H)


def law_ok(lengths, hi=HI, zmax=5.0):
    """Octave masses and, inside octaves 3.., the share of the lower half, all
    within zmax standard errors of the 1/x law."""
    n = lengths.size
    H = float(np.sum(1.0 / np.arange(1, hi + 1, dtype=np.float64)))
    j = 0
    while 2 ** j <= hi:
        a, b = 2 ** j, min(2 ** (j + 1) - 1, hi)
        p = harmonic_mass(a, b, H)
        c = int(np.sum((lengths >= a) & (lengths <= b)))
        if abs(c - n * p) > zmax * np.sqrt(n * p * (1 - p)):
            return False
        if j >= 3:
            mid = a + (b - a + 1) // 2
            q = harmonic_mass(a, mid - 1, H) / p  # lower half's share inside the octave
            lo = int(np.sum((lengths >= a) & (lengths < mid)))
            if abs(lo - c * q) > zmax * np.sqrt(c * q * (1 - q)):
                return False
        j += 1
    return True


def test_ragged_lengths_are_log_uniform():
    P = S.make_params("ragged", p_trunc=0.0)  # untruncated: the length drawn is the row's length
    lengths, _ = S.host_rows(P, N)
    assert lengths.min() >= 1 and lengths.max() <= HI
    assert law_ok(lengths.astype(np.int64))
    H = float(np.sum(1.0 / np.arange(1, HI + 1, dtype=np.float64)))
    mean = HI / H  # E[L] = sum_x x (1/x) / H
    assert abs(lengths.mean() - mean) < 0.02 * mean


def test_octave_uniform_law_is_rejected():
    rng = np.random.default_rng(0)
    j = rng.integers(0, 16, N)
    lo = 2 ** j
    hi = np.minimum(2 * lo - 1, HI)
    x = lo + (rng.random(N) * (hi - lo + 1)).astype(np.int64)
    assert not law_ok(x)
    # the 1/x law sampled by numpy passes the same checks
    H = np.cumsum(1.0 / np.arange(1, HI + 1, dtype=np.float64))
    y = 1 + np.searchsorted(H / H[-1], rng.random(N), side="right")
    assert law_ok(np.minimum(y, HI))


def test_ragged_workload_keeps_its_truncated_rows():
    P = S.make_params("ragged")
    full, _ = S.host_rows(S.make_params("ragged", p_trunc=0.0), 1024)
    got, _ = S.host_rows(P, 1024)
    assert np.all(got <= full)
    cut = np.mean(got < full)
    assert 0.02 < cut < 0.09  # 5 % of rows truncated at a uniform position
