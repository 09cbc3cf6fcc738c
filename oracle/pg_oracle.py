"""CPU oracle of the GRPO advantage and token-level clipped surrogate.

TEST INFRASTRUCTURE.  Only the tests and the smoke check may import this
module; the product path never does.  Plain numpy in float64.

The paper trains with GRPO in VeRL, 8 rollouts per prompt, and separate lower
and upper clip ratios of 0.2 and 0.28 (Sec. 4, "Training Framework"); it does
not write the objective out.  This oracle therefore follows the textbook
definitions, each a reading listed in the design notes:

* advantage of rollout i (GRPO, Shao et al. 2024, outcome supervision): the
  reward normalised within its group of G rollouts,
  A_i = (R_i - mean_g R) / std_g R, population standard deviation, A_i = 0 when
  every reward of the group is equal (no epsilon);
* ratio rho_t = exp(logp_t - logp_old_t) per generated token;
* clipped objective with separate lower and upper clip ratios (PPO clip with
  DAPO's "clip-higher", Yu et al. 2025):
  L_t = min(rho_t A, clip(rho_t, 1 - eps_low, 1 + eps_high) A);
* token-level mean over every generated token of the batch:
  J = sum_t L_t / N_tokens; the loss is -J; no KL or entropy term.

Everything is float64 from the float32 inputs: d = logp - logp_old (exact in
float64 for log-probabilities of similar magnitude), rho = exp(d), and the clip
decision is the definition itself: for A > 0 the clipped term is the minimum
exactly when rho > 1 + eps_high, for A < 0 exactly when rho < 1 - eps_low (at
equality both terms are equal; the unclipped one is taken).

Gradient of the loss with respect to logp_t:
  d(-J)/d logp_t = -A rho_t / N_tokens where the unclipped term is the minimum,
  else 0.
"""
from __future__ import annotations

import numpy as np


def advantages(reward, group_size: int) -> np.ndarray:
    """Group-normalised advantages (float64) of float rewards."""
    r = np.asarray(reward, dtype=np.float32).astype(np.float64)
    n = r.size
    assert n % group_size == 0
    out = np.zeros(n, np.float64)
    for g0 in range(0, n, group_size):
        x = r[g0: g0 + group_size]
        if np.all(x == x[0]):
            continue  # sigma = 0: A = 0
        mu = 0.0
        for v in x:
            mu = mu + v
        mu = mu / group_size
        ss = 0.0
        for v in x:
            ss = ss + (v - mu) * (v - mu)
        sigma = np.sqrt(ss / group_size)
        out[g0: g0 + group_size] = (x - mu) / sigma
    return out


def surrogate(logp, logp_old, starts, lengths, adv, eps_low: float, eps_high: float, n_tokens=None):
    """Loss, gradient and clip counts.

    logp, logp_old: float32 arrays; row i is [starts[i], starts[i] + lengths[i]).
    adv: advantage per row (the kernel stores it as float32, so pass that).
    n_tokens: N of the token-level mean, the generated tokens of the whole
    batch; by default the tokens of the rows given (pass the batch's N when
    the rows are a sample of a larger batch).
    Returns dict(loss, tokens, clip_high, clip_low, grad, clipped, d): grad is
    float64 with NaN outside the rows; clipped (bool) marks the tokens whose
    clipped term is the minimum; d is the float64 log-ratio (NaN outside)."""
    logp = np.asarray(logp, np.float32)
    logp_old = np.asarray(logp_old, np.float32)
    grad = np.full(logp.size, np.nan)
    dd = np.full(logp.size, np.nan)
    clipped_all = np.zeros(logp.size, bool)
    n_tok = int(np.sum(np.maximum(lengths, 0))) if n_tokens is None else int(n_tokens)
    hi, lo = 1.0 + float(eps_high), 1.0 - float(eps_low)
    total = 0.0
    clip_hi = clip_lo = 0
    for i in range(len(starts)):
        a = float(np.float32(adv[i]))
        s, n = int(starts[i]), int(lengths[i])
        if n <= 0:
            continue
        d = logp[s: s + n].astype(np.float64) - logp_old[s: s + n].astype(np.float64)
        rho = np.exp(d)
        if a > 0:
            clipped = rho > hi
            clip_hi += int(np.sum(clipped))
        elif a < 0:
            clipped = rho < lo
            clip_lo += int(np.sum(clipped))
        else:
            clipped = np.zeros(n, bool)
        # min(rho A, clip(rho) A): the clip bound where the decision says so
        L = np.where(clipped, (hi if a > 0 else lo) * a, rho * a)
        total += float(np.sum(L))
        grad[s: s + n] = np.where(clipped, 0.0, -a * rho / n_tok) if n_tok else 0.0
        clipped_all[s: s + n] = clipped
        dd[s: s + n] = d
    loss = -total / n_tok if n_tok else 0.0
    return dict(loss=loss, tokens=n_tok, clip_high=clip_hi, clip_low=clip_lo, grad=grad, clipped=clipped_all, d=dd)
