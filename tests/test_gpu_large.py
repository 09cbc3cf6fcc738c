"""The large workload (89,000 groups x 8 rows, mean 50.3k tokens: 3.6e10 tokens,
143 GB of int32) at full size, in the launch configuration the benchmark times,
compared with the oracle on every row.

The batch is generated on the device and run once; then every token is copied
back to the host in chunks of whole groups (pinned buffers), each chunk is
evaluated by the oracle on a host worker thread (the oracle is plain
single-threaded C; ctypes releases the interpreter lock around it), and all
712,000 rows are compared: integers bit-exact, floats as the float rounding of
the oracle's double values.  The host mirror of the generator is checked
against the device copy on a few rows, and properties that hold at any size
are checked on every row."""
import os
import queue
import threading
import time

import numpy as np
import pytest

from gpu_util import DEFAULT_COEF, compare, fetch, log
from oracle import oracle as O
from paper_2608_24658_amd import parason as PX
from paper_2608_24658_amd.synth import synth as S

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

G = S.GROUP_SIZE
CHUNK_TOKENS = 1 << 27  # about 0.35 s of oracle work per chunk


def host_workers():
    try:
        n = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def group_chunks(st_h, ln_h, chunk_tokens):
    """[(r0, r1)] row ranges of whole groups holding about chunk_tokens each."""
    n = st_h.size
    gtok = ln_h.astype(np.int64).reshape(-1, G).sum(1)
    cum = np.cumsum(gtok)
    out, g0 = [], 0
    while g0 < gtok.size:
        base = cum[g0 - 1] if g0 else 0
        g1 = int(np.searchsorted(cum, base + chunk_tokens, side="left")) + 1
        g1 = min(max(g1, g0 + 1), gtok.size)
        out.append((g0 * G, g1 * G))
        g0 = g1
    assert out[-1][1] == n
    return out


def oracle_streamed(tok_d, st_h, ln_h, tags, workers, chunk_tokens=CHUNK_TOKENS):
    """Oracle rows of a packed device batch (rows back to back from
    st_h[0]), streamed to the host chunk by chunk."""
    chunks = group_chunks(st_h, ln_h, chunk_tokens)
    ends = st_h + ln_h.astype(np.int64)
    cap = max(int(ends[r1 - 1] - st_h[r0]) for r0, r1 in chunks)
    nbuf = workers + 2
    bufs = [torch.empty(cap, dtype=torch.int32, pin_memory=True) for _ in range(nbuf)]
    free = queue.Queue()
    for i in range(nbuf):
        free.put(i)
    rows = np.zeros(st_h.size, O.ROW_DTYPE)
    todo = queue.Queue()
    errors = []

    def worker():
        while True:
            job = todo.get()
            if job is None:
                return
            b, r0, r1, m = job
            try:
                host = bufs[b].numpy()[:m]
                rows[r0:r1] = O.eval_rows(host, st_h[r0:r1] - st_h[r0], ln_h[r0:r1], tags)
            except Exception as e:  # reported by the main thread
                errors.append(e)
            free.put(b)

    threads = [threading.Thread(target=worker, daemon=True) for _ in range(workers)]
    for t in threads:
        t.start()
    t0 = time.time()
    for k, (r0, r1) in enumerate(chunks):
        lo, hi = int(st_h[r0]), int(ends[r1 - 1])
        b = free.get()
        bufs[b][: hi - lo].copy_(tok_d[lo:hi])  # device -> pinned host, synchronous
        todo.put((b, r0, r1, hi - lo))
        if k % 40 == 0:
            log("  chunk %d/%d (rows %d..%d) copied at %.1f s" % (k, len(chunks), r0, r1, time.time() - t0))
    for _ in threads:
        todo.put(None)
    for t in threads:
        t.join()
    if errors:
        raise errors[0]
    log("  oracle on %d rows in %d chunks, %d threads: %.1f s" % (st_h.size, len(chunks), workers, time.time() - t0))
    return rows


def test_large_workload_every_row(request):
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
    del out
    torch.cuda.empty_cache()  # the workspace

    # properties on every row
    assert np.array_equal(got["total"], ln_h)
    assert np.all(got["latency"] <= got["total"]) and np.all(got["latency"] > 0)
    assert np.all(got["n_subtask"] + got["n_trial"] <= got["total"] - 2)
    assert np.all(got["flags"] & PX.FLAG_VALID)  # every generated large row is complete
    assert np.all(np.isfinite(got["reward"]))
    assert np.all((got["reward"] == -1.0) == ((co_h == 0)))

    # the device tokens are the generator's (host mirror on a few rows)
    for r in (0, n // 3, n - 1):
        t = S.host_row_tokens(P, r, int(st_h[r]), int(ln_h[r]))
        d = tok_d[int(st_h[r]): int(st_h[r]) + int(ln_h[r])].cpu().numpy()
        assert np.array_equal(t, d), "row %d differs from the host mirror" % r

    # every row, compared in full with the oracle
    w = host_workers()
    log("case large: oracle on every row (%d host threads)" % w)
    rows = oracle_streamed(tok_d, st_h, ln_h, S.CONTIGUOUS_TAGS, w)
    c = DEFAULT_COEF
    R, rs, rt, eta = O.group_reward(rows, co_h, G, c["alpha"], c["beta_subtask"], c["beta_trial"],
                                    c["rho"], c["rho_clip"])
    n_exact = compare(got, rows, R, rs, rt, eta, what="large, every row")
    assert n_exact == n
    log("large: %d rows, %d tokens; every row matches the oracle (latency sum %d, Subtask %d, Trial %d)" % (
        n, total, int(rows["latency"].astype(np.int64).sum()), int(rows["n_subtask"].astype(np.int64).sum()),
        int(rows["n_trial"].astype(np.int64).sum())))
    del tok_d
    torch.cuda.empty_cache()


def max_row(tags, rng, extra=0):
    """A row of INT32_MAX tokens: <think>, a block straddling position 2^30,
    a block just before </think>, then 100 answer tokens; and its accounting
    in closed form.  The buffer has `extra` more tokens after the row."""
    L = 2**31 - 1
    tok = np.full(L + extra, 7, np.int32)  # one text id; random text ids around the blocks and the ends
    for lo in (0, 2**30 - 70000, L - 70000):
        w = rng.integers(0, 150000, size=65536).astype(np.int32)
        tok[lo: lo + w.size] = np.where(np.isin(w, tags), 7, w)

    def place(off, names):
        import grammar_pins as GP

        for i, c in enumerate(GP.parse_names(names)):
            if c:
                tok[off + i] = tags[c - 1]
        return len(GP.parse_names(names))

    place(0, "think")
    n_a = place(2**30 - 7, "Par Out Sub t3 /Sub Tri t1 /Tri /Out Thr t5000 /Thr Thr t10 /Thr /Par")
    n_b = place(L - 141, "Par Out Tri t2 /Tri Tri t2 /Tri /Out Thr t7 /Thr Thr t9 /Thr /Par")
    place(L - 101, "/think")
    assert (n_a, n_b) == (5026, 32)
    # block A: lat = 1 + 10 + max(5002, 12) + 1 = 5014 of 5026 tokens (saves 12);
    # thread 0 pairs with the Subtask entry (5002 tokens), thread 1 with the Trial (12);
    # block B: lat = 1 + 10 + max(9, 11) + 1 = 23 of 32 tokens (saves 9), 20 Trial tokens
    expect = dict(total=L, latency=L - 21, n_subtask=5002, n_trial=32, n_blocks=2, max_depth=1,
                  first_error_pos=-1, flags=PX.FLAG_VALID | PX.FLAG_TRIGGERED)
    return tok, expect


def test_rows_of_int32_max_tokens():
    """Rows at the largest length the interface takes (INT32_MAX tokens):
    one complete, overlapping prefixes of it (valid after </think>, truncated
    before it), a copy that starts one token late (misaligned, invalid at 0),
    and four small rows; closed forms and the oracle."""
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    dev = torch.device("cuda:0")
    rng = np.random.default_rng(17)
    tags = S.CONTIGUOUS_TAGS
    log("case int32-max rows: host row")
    P = S.make_params("tiny")
    tok_s, st_s, ln_s, co_s = S.host_batch(P, 4)
    tokens, expect = max_row(tags, rng, extra=tok_s.size)
    L = expect["total"]
    tokens[L:] = tok_s
    starts = np.array([0, 0, 1, 0] + list(st_s + L), np.int64)
    lengths = np.array([L, L - 200, L - 1, L - 50] + list(ln_s), np.int32)
    correct = np.array([1, 1, 1, 0] + list(co_s), np.uint8)
    px = PX.Parason(tags, group_size=G, **DEFAULT_COEF)
    log("case int32-max rows: run (%d tokens in the buffer)" % tokens.size)
    tok_d = torch.from_numpy(tokens).to(dev)
    out = px.run(tok_d, torch.from_numpy(starts).to(dev), torch.from_numpy(lengths).to(dev),
                 torch.from_numpy(correct).to(dev))
    torch.cuda.synchronize()
    got = fetch(out)
    del tok_d, out
    torch.cuda.empty_cache()
    for k, v in expect.items():
        assert int(got[k][0]) == v, (k, int(got[k][0]), v)
    assert int(got["first_error_pos"][1]) == L - 200 and got["flags"][1] == PX.FLAG_TRUNCATED
    assert int(got["latency"][1]) == L - 200
    assert int(got["first_error_pos"][2]) == 0 and got["flags"][2] == 0
    assert int(got["latency"][3]) == L - 50 - 21 and got["flags"][3] == expect["flags"]
    assert int(got["saved"][0]) == 21
    log("case int32-max rows: oracle")
    rows = O.eval_rows(tokens, starts, lengths, tags)
    c = DEFAULT_COEF
    R, rs, rt, eta = O.group_reward(rows, correct, G, c["alpha"], c["beta_subtask"], c["beta_trial"], c["rho"],
                                    c["rho_clip"])
    compare(got, rows, R, rs, rt, eta, what="int32-max rows")
    log("int32-max rows match")
