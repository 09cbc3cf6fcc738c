"""Pins of the CPU oracle against what the paper and the mathematics fix.

Every check here compares the oracle with something other than itself: the
grammar via an Earley recognizer, the latency via a fork/join DAG longest path,
closed forms, invariants, the paper's printed numbers (Table 5) and a hand
computed worked example (the repaired Figure 3).
"""
import json
import os
import random

import numpy as np
import pytest

import grammar_pins as G
from oracle import oracle as O

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")
TAGS = np.arange(151936 - 12, 151936, dtype=np.int32)  # contiguous ids at the top of the vocabulary
SCATTERED = np.array([5, 900, 17, 151000, 3, 77777, 42, 1000, 2**31 - 1, 123456, 64, 8], dtype=np.int32)


def run(classes, tags=TAGS, text_id=7):
    return O.eval_stream(G.to_tokens(classes, tags, text_id), tags)


def expected_depth(classes):
    d = m = 0
    for c in classes:
        if c == G.PAR:
            d += 1
            m = max(m, d)
        elif c == G.END_PAR:
            d -= 1
    return m


def independent_row(classes):
    """Expected accounting of a valid stream from the pins only."""
    lat, _ = G.dag_latency(classes)
    types = G.thread_types(classes)
    return dict(
        total=len(classes),
        latency=lat,
        n_subtask=sum(1 for t in types if t == 1),
        n_trial=sum(1 for t in types if t == 2),
        n_blocks=classes.count(G.PAR),
        max_depth=expected_depth(classes),
    )


def check_row(r, classes):
    exp = independent_row(classes)
    for k, v in exp.items():
        assert int(r[k]) == v, (k, int(r[k]), v, " ".join(G.NAMES[c] for c in classes))


# --------------------------------------------------------------------------- grammar


@pytest.mark.parametrize("tags", [TAGS, SCATTERED], ids=["contiguous", "scattered"])
def test_every_valid_string_up_to_20(tags):
    strings = G.enumerate_valid(20)
    assert len(strings) > 10000
    for s in strings:
        s = list(s)
        r = run(s, tags)
        assert r["flags"] & O.F_VALID, s
        assert r["first_error_pos"] == -1
        check_row(r, s)


def _mutations(s, rng, k):
    out = []
    n = len(s)
    for _ in range(k):
        op = rng.randrange(3)
        if op == 0 and n:
            i = rng.randrange(n)
            out.append(s[:i] + [rng.randrange(13)] + s[i + 1:])
        elif op == 1 and n:
            i = rng.randrange(n)
            out.append(s[:i] + s[i + 1:])
        else:
            i = rng.randrange(n + 1)
            out.append(s[:i] + [rng.randrange(13)] + s[i:])
    return out


def test_validity_and_first_error_match_earley_on_mutations():
    rng = random.Random(1234)
    strings = [list(s) for s in G.enumerate_valid(20)]
    sample = rng.sample(strings, 1500)
    cases = []
    for s in sample:
        cases += _mutations(s, rng, 4)
        cases.append(s[: rng.randrange(len(s) + 1)])  # truncation
    n_invalid = 0
    for s in cases:
        ok, err = G.earley(s)
        r = run(s)
        assert bool(r["flags"] & O.F_VALID) == ok, s
        assert int(r["first_error_pos"]) == err, (s, int(r["first_error_pos"]), err)
        assert bool(r["flags"] & O.F_TRUNCATED) == (not ok and err == len(s))
        if ok:
            check_row(r, s)
        else:
            n_invalid += 1
            assert (r["latency"], r["n_subtask"], r["n_trial"], r["n_blocks"], r["max_depth"]) == (len(s), 0, 0, 0, 0)
            assert not r["flags"] & O.F_TRIGGERED
    assert n_invalid > 3000


def test_random_short_strings_match_earley():
    rng = random.Random(99)
    alphabet = list(range(13))
    for _ in range(20000):
        n = rng.randrange(0, 9)
        s = [G.THINK] + [rng.choice(alphabet) for _ in range(n)] if rng.random() < 0.8 else [rng.choice(alphabet) for _ in range(n)]
        ok, err = G.earley(s)
        r = run(s)
        assert bool(r["flags"] & O.F_VALID) == ok, s
        assert int(r["first_error_pos"]) == err, s


def test_empty_and_degenerate_streams():
    r = run([])
    assert r["flags"] == O.F_TRUNCATED and r["first_error_pos"] == 0 and r["total"] == 0 and r["latency"] == 0
    r = run([G.THINK])
    assert r["flags"] == O.F_TRUNCATED and r["first_error_pos"] == 1
    r = run([G.TEXT, G.THINK, G.END_THINK])  # nothing may precede <think>
    assert r["flags"] == 0 and r["first_error_pos"] == 0
    r = run([G.THINK, G.END_THINK])
    assert r["flags"] == O.F_VALID and r["latency"] == 2
    r = run([G.THINK, G.END_THINK, G.TEXT, G.TEXT])  # the answer after </think>
    assert r["flags"] == O.F_VALID and r["latency"] == 4
    r = run([G.THINK, G.END_THINK, G.TEXT, G.THINK])  # a tag after </think>
    assert r["flags"] == 0 and r["first_error_pos"] == 3
    # empty entry text: T is non-empty
    s = G.parse_names("think Par Out Sub /Sub")
    r = run(s)
    assert r["flags"] == 0 and r["first_error_pos"] == 4


def test_count_mismatch_flag_and_surplus_threads_untyped():
    s = G.parse_names("think Par Out Sub t3 /Sub /Out Thr t4 /Thr Thr t5 /Thr /Par /think")
    r = run(s)
    assert r["flags"] == O.F_VALID | O.F_TRIGGERED | O.F_COUNT_MISMATCH
    assert r["n_subtask"] == 6 and r["n_trial"] == 0  # second thread has no entry
    check_row(r, s)
    s = G.parse_names("think Par Out Tri t3 /Tri Tri t1 /Tri /Out Thr t4 /Thr /Par /think")
    r = run(s)
    assert r["flags"] == O.F_VALID | O.F_TRIGGERED | O.F_COUNT_MISMATCH
    assert r["n_trial"] == 6


# --------------------------------------------------------------------------- worked example


def test_repaired_figure3_golden():
    g = json.load(open(os.path.join(GOLDEN, "fig3_repaired.json")))
    s = G.parse_names(g["stream"])
    for tags in (TAGS, SCATTERED):
        r = run(s, tags)
        for k, v in g["expected"].items():
            assert int(r[k]) == v, (k, int(r[k]), v)
    # the independent pins agree with the hand computation as well
    exp = independent_row(s)
    for k, v in exp.items():
        assert g["expected"][k] == v


def test_figure3_as_printed_is_not_in_the_language():
    # Inner blocks without threads and a second </Outlines> (Figure 3) are rejected.
    s = G.parse_names("think t5 Par Out Sub t3 /Sub Sub t3 /Sub Sub t3 /Sub Thr t1 Par Out Tri t4 /Tri /Out /Par /Thr /Out /Out /Par t2 /think")
    r = run(s)
    ok, err = G.earley(s)
    assert not ok and not (r["flags"] & O.F_VALID) and r["first_error_pos"] == err


# --------------------------------------------------------------------------- closed forms


def single_block(main_a, main_b, entries, bodies, kind=G.TRI):
    close = G.END_TRI if kind == G.TRI else G.END_SUB
    s = [G.THINK] + [G.TEXT] * main_a + [G.PAR, G.OUT]
    for e in entries:
        s += [kind] + [G.TEXT] * e + [close]
    s += [G.END_OUT]
    for b in bodies:
        s += [G.THR] + [G.TEXT] * b + [G.END_THR]
    s += [G.END_PAR] + [G.TEXT] * main_b + [G.END_THINK]
    return s


def test_single_block_closed_form():
    rng = random.Random(5)
    for _ in range(300):
        k = rng.randint(1, 6)
        entries = [rng.randint(1, 9) for _ in range(k)]
        bodies = [rng.randint(0, 40) for _ in range(k)]
        a, b = rng.randint(0, 30), rng.randint(0, 30)
        kind = rng.choice([G.SUB, G.TRI])
        s = single_block(a, b, entries, bodies, kind)
        r = run(s)
        lat = (a + b) + 2 + 2 + (2 + sum(2 + e for e in entries)) + max(2 + x for x in bodies)
        assert r["latency"] == lat
        assert r["total"] == len(s)
        branch = sum(2 + x for x in bodies)
        assert r["n_subtask" if kind == G.SUB else "n_trial"] == branch
        assert r["n_trial" if kind == G.SUB else "n_subtask"] == 0
        assert r["total"] - r["latency"] == branch - max(2 + x for x in bodies)


def test_no_parallel_means_sequential():
    for n in range(0, 50, 7):
        s = [G.THINK] + [G.TEXT] * n + [G.END_THINK] + [G.TEXT] * (n // 2)
        r = run(s)
        assert r["latency"] == r["total"] == len(s)
        assert r["n_blocks"] == 0 and r["flags"] == O.F_VALID


def test_table5_identities():
    """Streams realising each Table 5 row reproduce its printed acceleration and saved tokens."""
    g = json.load(open(os.path.join(GOLDEN, "table5_identities.json")))
    for row in g["rows"]:
        gen, lat_t = row["generated"], row["latency"]
        saved = gen - lat_t
        # two equal threads: total - latency = lat(W) = saved
        body = saved - 2
        entries = [1, 1]
        fixed = 2 + 1 + (2 + 3 + 3) + 1 + 2 * saved
        main = gen - fixed
        s = single_block(main, 0, entries, [body, body])
        rows = O.eval_rows(np.array(G.to_tokens(s, TAGS)), np.array([0]), np.array([len(s)]), TAGS)
        r = rows[0]
        assert r["total"] == gen and r["latency"] == lat_t
        assert round(r["total"] / r["latency"], 2) == row["acceleration"]
        assert r["total"] - r["latency"] == row["saved"]
        _, _, _, eta = O.group_reward(rows, [1], 1, 0, 0, 0, 1.0, 1.0)
        assert abs(1.0 / (1.0 - eta[0]) - row["acceleration"]) < 0.005
        accel, saved_o = O.row_acceleration(rows)
        assert round(accel[0], 2) == row["acceleration"] and saved_o[0] == row["saved"]


def test_row_acceleration_definitions():
    rng = np.random.default_rng(3)
    rows = np.zeros(200, dtype=O.ROW_DTYPE)
    rows["total"] = rng.integers(0, 60000, 200)
    rows["latency"] = np.minimum(rows["total"], rng.integers(1, 60000, 200))
    rows["total"][:3] = 0
    rows["latency"][:3] = 0
    accel, saved = O.row_acceleration(rows)
    assert np.all(accel[:3] == 1.0) and np.all(saved[:3] == 0)
    _, _, _, eta = O.group_reward(rows, np.ones(200, np.uint8), 1, 0, 0, 0, 1.0, 1.0)
    # acceleration = 1 / (1 - eta) and saved = eta * total (eta of Sec. 3.3)
    assert np.allclose(accel, 1.0 / (1.0 - eta), rtol=1e-12)
    assert np.allclose(saved, eta * rows["total"], rtol=0, atol=1e-6)


# --------------------------------------------------------------------------- invariants on random trees


def random_body(rng, depth, budget):
    items = []
    for _ in range(rng.randint(0, 3)):
        if depth < 4 and rng.random() < 0.45:
            items.append(random_block(rng, depth + 1, budget))
        else:
            items.append(rng.randint(1, budget))
    return items


def random_block(rng, depth, budget):
    kind = rng.choice([G.SUB, G.TRI])
    n_e = rng.randint(1, 4)
    n_t = n_e if rng.random() < 0.85 else rng.randint(1, 5)
    entries = [(rng.choice([G.SUB, G.TRI]) if rng.random() < 0.2 else kind, rng.randint(1, budget)) for _ in range(n_e)]
    threads = [random_body(rng, depth, budget) for _ in range(n_t)]
    return ("P", entries, threads)


def render_body(items, out):
    for it in items:
        if isinstance(it, int):
            out += [G.TEXT] * it
        else:
            _, entries, threads = it
            out += [G.PAR, G.OUT]
            for kind, e in entries:
                out += [kind] + [G.TEXT] * e + [G.END_SUB if kind == G.SUB else G.END_TRI]
            out += [G.END_OUT]
            for t in threads:
                out.append(G.THR)
                render_body(t, out)
                out.append(G.END_THR)
            out.append(G.END_PAR)
    return out


def blocks_of(items, acc):
    for it in items:
        if not isinstance(it, int):
            acc.append(it)
            for t in it[2]:
                blocks_of(t, acc)
    return acc


def test_invariants_on_random_trees():
    rng = random.Random(2024)
    streams = []
    for _ in range(400):
        body = random_body(rng, 0, 12)
        s = [G.THINK] + render_body(body, []) + [G.END_THINK] + [G.TEXT] * rng.randint(0, 5)
        streams.append((body, s))
    toks = np.concatenate([np.array(G.to_tokens(s, TAGS), np.int32) for _, s in streams])
    lens = np.array([len(s) for _, s in streams], np.int32)
    starts = np.concatenate([[0], np.cumsum(lens)[:-1]]).astype(np.int64)
    rows = O.eval_rows(toks, starts, lens, TAGS)
    for (body, s), r in zip(streams, rows):
        assert r["flags"] & O.F_VALID
        check_row(r, s)
        lat, per_block = G.dag_latency(s)
        # total - latency = sum over all blocks of (sum_k lat W_k - max_k lat W_k)
        assert r["total"] - r["latency"] == sum(sum(b) - max(b) for b in per_block)
        blocks = blocks_of(body, [])
        one_thread_everywhere = all(len(b[2]) == 1 for b in blocks)
        assert (r["latency"] == r["total"]) == one_thread_everywhere
        assert r["latency"] <= r["total"]
        assert r["n_subtask"] + r["n_trial"] <= r["total"] - 2
        mismatch = any(len(b[1]) != len(b[2]) for b in blocks)
        assert bool(r["flags"] & O.F_COUNT_MISMATCH) == mismatch
        assert bool(r["flags"] & O.F_TRIGGERED) == (len(blocks) > 0)


def test_deep_nesting_does_not_overflow():
    depth = 20000
    s = [G.THINK]
    for _ in range(depth):
        s += [G.PAR, G.OUT, G.SUB, G.TEXT, G.END_SUB, G.END_OUT, G.THR]
    s += [G.TEXT]
    for _ in range(depth):
        s += [G.END_THR, G.END_PAR]
    s += [G.END_THINK]
    r = run(s)
    assert r["flags"] == O.F_VALID | O.F_TRIGGERED
    assert r["max_depth"] == depth and r["n_blocks"] == depth
    assert r["latency"] == r["total"]  # one thread per block
    # everything from the first <Thread> (index 7) to the outermost </Thread>
    # (third token from the end, before </Parallel> </think>) is Subtask
    first_thr = 1 + 6
    last_thr = len(s) - 3
    assert r["n_subtask"] == last_thr - first_thr + 1


# --------------------------------------------------------------------------- reward


def _rows(lat, total, sub, tri, valid=True):
    rows = np.zeros(len(lat), dtype=O.ROW_DTYPE)
    rows["latency"], rows["total"], rows["n_subtask"], rows["n_trial"] = lat, total, sub, tri
    rows["flags"] = O.F_VALID if valid else 0
    return rows


def test_reward_incorrect_is_minus_one():
    rng = np.random.default_rng(0)
    total = rng.integers(1, 10000, 16)
    rows = _rows(rng.integers(1, total + 1), total, rng.integers(0, total // 2 + 1), rng.integers(0, total // 2 + 1))
    R, *_ = O.group_reward(rows, np.zeros(16), 8, 0.1, 0.05, 0.1, 0.5, 0.25)
    assert np.all(R == -1.0)


def test_reward_constant_group_closed_form():
    for rho, clip in [(0.5, 0.25), (2.0, 0.1), (0.1, 1.0)]:
        rows = _rows([700] * 8, [1000] * 8, [100] * 8, [300] * 8)
        R, _, _, eta = O.group_reward(rows, np.ones(8), 8, 0.1, 0.05, 0.1, rho, clip)
        assert np.all(eta == 1 - 700 / 1000)
        # exact in real arithmetic; a few double roundings apart in floating point
        np.testing.assert_allclose(R, 1 + 2 * min(rho * (1 - 0.7), clip), rtol=0, atol=1e-15)


def test_equal_ratios_with_different_denominators_normalise_to_zero():
    # 1/3 and 2/6 are the same ratio: sigma is 0 exactly, so z = 0.
    rows = _rows([5, 10, 15, 20, 5, 10, 15, 20], [30, 60, 90, 120, 30, 60, 90, 120], [10, 20, 30, 40, 10, 20, 30, 40], [0] * 8)
    R, *_ = O.group_reward(rows, np.ones(8), 8, 0.0, 1.0, 0.0, 0.0, 0.0)
    assert np.all(R == 1.0)


def test_zscores_match_numpy_and_normalise():
    rng = np.random.default_rng(7)
    G_ = 8
    n = 64 * G_
    total = rng.integers(50, 60000, n)
    lat = np.array([rng.integers(t // 3, t + 1) for t in total])
    sub = np.array([rng.integers(0, t // 2) for t in total])
    tri = np.array([rng.integers(0, t - s) for t, s in zip(total, sub)])
    rows = _rows(lat, total, sub, tri)
    ones = np.ones(n)
    # alpha = 1, everything else 0: R = 1 - 2 z_T
    R, rs, rt, eta = O.group_reward(rows, ones, G_, 1.0, 0.0, 0.0, 0.0, 0.0)
    zT = (1.0 - R) / 2.0
    Rs, *_ = O.group_reward(rows, ones, G_, 0.0, 1.0, 0.0, 0.0, 0.0)
    zs = (Rs - 1.0) / 2.0
    Rr, *_ = O.group_reward(rows, ones, G_, 0.0, 0.0, 1.0, 0.0, 0.0)
    zr = (Rr - 1.0) / 2.0
    for z, x in ((zT, lat.astype(np.float64)), (zs, sub / total), (zr, tri / total)):
        xg = x.reshape(-1, G_)
        ref = (xg - xg.mean(axis=1, keepdims=True)) / xg.std(axis=1, ddof=0, keepdims=True)
        np.testing.assert_allclose(z.reshape(-1, G_), ref, rtol=1e-12, atol=1e-12)
        zg = z.reshape(-1, G_)
        np.testing.assert_allclose(zg.sum(axis=1), 0.0, atol=1e-12)
        np.testing.assert_allclose((zg ** 2).sum(axis=1), G_, rtol=1e-12)
    np.testing.assert_array_equal(rs, sub / total)
    np.testing.assert_array_equal(rt, tri / total)
    np.testing.assert_allclose(eta, 1 - lat / total, rtol=0, atol=1e-15)
    # the reward is affine in (alpha, beta_s, beta_r)
    Rall, *_ = O.group_reward(rows, ones, G_, 0.3, 0.2, 0.1, 0.0, 0.0)
    np.testing.assert_allclose(Rall, -1 + 2 * (1 - 0.3 * zT + 0.2 * zs + 0.1 * zr), rtol=0, atol=1e-12)


def test_invalid_rollout_policy():
    rows = _rows([10] * 8, [10] * 8, [0] * 8, [0] * 8, valid=False)
    R, *_ = O.group_reward(rows, np.ones(8), 8, 0.1, 0.0, 0.0, 0.5, 0.25)
    assert np.all(R == -1.0)
    R, *_ = O.group_reward(rows, np.ones(8), 8, 0.1, 0.0, 0.0, 0.5, 0.25, cfg_flags=O.CFG_INVALID_KEEPS_CORRECTNESS)
    assert np.all(R == 1.0)  # z = 0, eta = 0


def test_group_size_must_divide():
    rows = _rows([1] * 6, [1] * 6, [0] * 6, [0] * 6)
    with pytest.raises(ValueError):
        O.group_reward(rows, np.ones(6), 4, 0, 0, 0, 0, 0)


# --------------------------------------------------------------------------- batch metrics


def test_batch_metrics_table5_and_table4_definitions():
    """Batch metrics on rows that realise Table 5's averages: acceleration =
    generated / latency tokens and saved = generated - latency as printed."""
    g = json.load(open(os.path.join(GOLDEN, "table5_identities.json")))
    for row in g["rows"]:
        gen, lat_t = row["generated"], row["latency"]
        saved = gen - lat_t
        body = saved - 2
        s = single_block(gen - (2 + 1 + (2 + 3 + 3) + 1 + 2 * saved), 0, [1, 1], [body, body])
        one = np.array(G.to_tokens(s, TAGS), np.int32)
        n = 6  # a few identical rows plus two sequential rows
        seq = np.array(G.to_tokens([G.THINK] + [G.TEXT] * 98 + [G.END_THINK], TAGS), np.int32)
        toks = np.concatenate([one] * n + [seq, seq])
        lens = np.array([one.size] * n + [seq.size] * 2, np.int32)
        starts = np.concatenate([[0], np.cumsum(lens)[:-1]]).astype(np.int64)
        rows = O.eval_rows(toks, starts, lens, TAGS)
        correct = np.array([1, 0, 1, 1, 0, 1, 1, 0], np.uint8)
        R, *_ = O.group_reward(rows, correct, 8, 0.1, 0.0, 0.1, 0.5, 0.25)
        m = O.batch_metrics(rows, correct, R)
        assert m["rows"] == 8 and m["valid"] == 8 and m["triggered"] == 6 and m["correct"] == 5
        assert m["trigger_ratio"] == 6 / 8
        assert m["sum_total"] == n * gen + 200 and m["sum_latency"] == n * lat_t + 200
        assert m["acceleration"] == (n * gen + 200) / (n * lat_t + 200)
        assert m["mean_saved"] == n * saved / 8
        assert m["accuracy"] == 5 / 8
        assert abs(m["mean_reward"] - R.mean()) < 1e-15
        # the identical rows alone reproduce the printed ratio and saved tokens
        m6 = O.batch_metrics(rows[:n], correct[:n], R[:n])
        assert round(m6["acceleration"], 2) == row["acceleration"] and m6["mean_saved"] == row["saved"]
        assert m6["trial_share"] == 2 * saved / gen and m6["subtask_share"] == 0


def test_batch_stats_is_one_group_over_the_batch():
    rng = np.random.default_rng(3)
    n = 40
    rows = np.zeros(n, dtype=O.ROW_DTYPE)
    rows["total"] = rng.integers(10, 1000, n)
    rows["latency"] = [rng.integers(1, t + 1) for t in rows["total"]]
    rows["n_subtask"] = [rng.integers(0, t // 2) for t in rows["total"]]
    rows["n_trial"] = [rng.integers(0, t // 2) for t in rows["total"]]
    rows["flags"] = O.F_VALID
    ones = np.ones(n)
    a = O.group_reward(rows, ones, 8, 0.2, 0.1, 0.05, 0.5, 0.25, O.CFG_BATCH_STATS)
    b = O.group_reward(rows, ones, n, 0.2, 0.1, 0.05, 0.5, 0.25)
    for x, y in zip(a, b):
        np.testing.assert_array_equal(x, y)
    # z over the batch: alpha = 1 isolates z_T; it matches numpy over all rows
    R, *_ = O.group_reward(rows, ones, 8, 1.0, 0.0, 0.0, 0.0, 0.0, O.CFG_BATCH_STATS)
    x = rows["latency"].astype(np.float64)
    np.testing.assert_allclose((1 - R) / 2, (x - x.mean()) / x.std(), rtol=1e-12, atol=1e-12)
