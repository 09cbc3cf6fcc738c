#!/usr/bin/env python3
"""Benchmark of the Parason accounting/reward hot path on one MI355X.

One step = one parason_run over the whole resident batch: segment plan, tag
scan of every token, per-row grammar automaton, group normalisation and the
reward of Definition 3.1.  The default workload is the large one: 89,000
prompts x 8 rollouts, rows of 25,150-75,450 tokens (mean 50.3k, the hard rows
of Table 5): 3.58e10 int32 tokens, 143 GB, resident in HBM before timing.

Prints one JSON line (rank 0, N = 1).  `value` is tokens per second of the
whole step.  `roofline` is for the dominant kernel (scan_rows: the token scan, which also
runs the grammar automaton of every row it holds whole), timed with HIP events
recorded around its launch on the run's stream; its achieved rate uses
algorithmic bytes: 4 B per token + 12 B per row read (start, length) + 32 B
per row written (the eight integer outputs).
`cpu_baseline` times the CPU oracle (single-threaded C) on a bounded sample of
the same rows.
"""
from __future__ import annotations

import argparse
import ctypes
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0  # MI355X HBM3E peak, GB/s
PROFILE_TRAFFIC = os.path.join(ROOT, "profiles", "scan_rows_large_traffic.json")


def log(msg):
    print(msg, file=sys.stderr, flush=True)


class HipEvents:
    """hipEvent_t pairs through the HIP runtime (the stream is the run's stream)."""

    def __init__(self):
        self.hip = ctypes.CDLL("libamdhip64.so")
        self.hip.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
        self.hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p, ctypes.c_void_p]
        self.hip.hipEventSynchronize.argtypes = [ctypes.c_void_p]
        self.hip.hipEventDestroy.argtypes = [ctypes.c_void_p]
        self.hip.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]

    def record(self, e, stream):
        rc = self.hip.hipEventRecord(e, ctypes.c_void_p(stream))
        if rc != 0:
            raise RuntimeError("hipEventRecord failed: %d" % rc)

    def create(self):
        e = ctypes.c_void_p()
        rc = self.hip.hipEventCreate(ctypes.byref(e))
        if rc != 0:
            raise RuntimeError("hipEventCreate failed: %d" % rc)
        return e

    def elapsed_ms(self, a, b):
        self.hip.hipEventSynchronize(b)
        ms = ctypes.c_float()
        rc = self.hip.hipEventElapsedTime(ctypes.byref(ms), a, b)
        if rc != 0:
            raise RuntimeError("hipEventElapsedTime failed: %d" % rc)
        return float(ms.value)


def cpu_baseline(tokens_d, starts_h, lengths_h, correct_h, tag_ids, coef, budget_s=12.0):
    """Time the CPU oracle on the first groups of the batch (copied to the host
    outside the timed region), sized for about budget_s seconds of CPU work.
    Returns the baseline record and the oracle's results on those rows (for
    the parity check against the GPU outputs)."""
    import numpy as np

    from oracle import oracle as O

    G = 8

    def sample(n_groups):
        n = n_groups * G
        lo, hi = int(starts_h[0]), int(starts_h[n - 1] + lengths_h[n - 1])
        toks = tokens_d[lo:hi].cpu().numpy()
        return toks, (starts_h[:n] - lo).astype(np.int64), lengths_h[:n].copy(), correct_h[:n].copy()

    def timed(toks, st, ln, co):
        t0 = time.perf_counter()
        rows = O.eval_rows(toks, st, ln, tag_ids)
        res = O.group_reward(rows, co, G, coef["alpha"], coef["beta_subtask"], coef["beta_trial"], coef["rho"],
                             coef["rho_clip"])
        return time.perf_counter() - t0, rows, res

    probe = sample(4)
    dt, _, _ = timed(*probe)
    rate = probe[0].size / max(dt, 1e-6)
    want = budget_s * rate
    per_group = probe[0].size / 4
    n_groups = int(max(4, min(len(starts_h) // G, want / per_group)))
    toks, st, ln, co = sample(n_groups)
    dt, rows, (R, rs, rt, eta) = timed(toks, st, ln, co)
    accel, saved = O.row_acceleration(rows)
    rec = {
        "value": toks.size / dt,
        "unit": "tokens/s",
        "cores": 1,
        "kind": "oracle",
        "sample": "first %d groups (%d rows, %d tokens) of the same workload, copied to the host; %.1f s "
                  "single-threaded" % (n_groups, n_groups * G, toks.size, dt),
        "rows_per_s": n_groups * G / dt,
        "host": host_cpu(),
    }
    return rec, dict(rows=rows, reward=R, r_subtask=rs, r_trial=rt, eta=eta, accel=accel, saved=saved)


def parity_of(out, ref):
    """Rows of the GPU outputs `out` (device tensors of the last timed step)
    that differ from the oracle's results `ref` on the rows ref covers (the
    first rows of the batch): integers and flags exactly, float outputs as the
    float rounding of the oracle's double values."""
    import numpy as np

    from paper_2608_24658_amd import parason as PX

    rows = ref["rows"]
    m = rows.size
    bad = np.zeros(m, bool)
    for k in PX.INT_FIELDS:
        bad |= out[k][:m].cpu().numpy() != rows[k]
    bad |= out["flags"][:m].cpu().numpy().view(np.uint32) != rows["flags"]
    for k in ("reward", "r_subtask", "r_trial", "eta", "accel"):
        bad |= out[k][:m].cpu().numpy() != ref[k].astype(np.float32)
    bad |= out["saved"][:m].cpu().numpy() != ref["saved"]
    return {"rows_checked": int(m), "mismatches": int(bad.sum()),
            "compared": "every integer output and flag exactly; reward, R_subtask, R_trial, eta, acceleration as "
                        "the float rounding of the oracle's double values; the cpu_baseline sample's rows against "
                        "the last timed step"}


def host_cpu():
    """The host's CPU model and the threads this process may run on."""
    import os

    model = "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        threads = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        threads = os.cpu_count()
    return {"cpu_model": model, "threads_available": threads}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="large", choices=["tiny", "small", "typical", "large", "ragged"])
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-typical-batch", action="store_true",
                    help="skip the typical-workload step timed after the large one (for profiler runs, so that "
                         "per-kernel averages cover one workload)")
    ap.add_argument("--cpu-budget", type=float, default=12.0)
    ap.add_argument("--step", default="accounting", choices=["accounting", "pg", "decode", "fork"],
                    help="accounting: the hot path (default); pg: the policy-gradient step that consumes its "
                         "rewards; decode: the grammar-constrained decode step of the rollouts; fork: fork/join "
                         "packing of worker contexts for tool-call execution")
    ap.add_argument("--decode-batch", type=int, default=1024)
    ap.add_argument("--calibrate-copy", action="store_true",
                    help="only run a plain device-to-device copy of 4 GiB (HBM counter calibration)")
    ap.add_argument("--traffic-summary", metavar="DIR",
                    help="only summarise the four rocprofv3 --pmc runs under DIR (prof_fetch, prof_write, "
                         "prof_copy_fetch, prof_copy_write) into the scan's traffic record under profiles/")
    args = ap.parse_args()

    if args.traffic_summary:
        traffic_summary(args.traffic_summary)
        return

    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path "
              "(groups would shard across GPUs with no exchange). Use --gpus 1.",
              file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    if args.calibrate_copy:
        # known traffic: 4 GiB read + 4 GiB written per copy
        x = torch.ones(1 << 30, dtype=torch.int32, device="cuda:0")
        y = torch.empty_like(x)
        for _ in range(3):
            y.copy_(x)
        torch.cuda.synchronize()
        print(json.dumps({"calibration": "copy", "bytes_read": 4 << 30, "bytes_written": 4 << 30, "launches": 3}))
        return

    from paper_2608_24658_amd import parason as PX
    from paper_2608_24658_amd.synth import synth as S

    if args.step == "pg":
        return bench_pg(args)
    if args.step == "decode":
        return bench_decode(args)
    if args.step == "fork":
        return bench_fork(args)

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    G = S.GROUP_SIZE
    coef = dict(alpha=0.1, beta_subtask=0.0, beta_trial=0.1, rho=0.5, rho_clip=0.25)

    P = S.make_params(args.workload)
    n = S.n_rows_of(args.workload)
    log("generating %s: %d rows" % (args.workload, n))
    t0 = time.time()
    tokens, starts, lengths, correct = S.device_batch(P, n, device=dev)
    torch.cuda.synchronize()
    n_tok = int(tokens.numel())
    log("generated %d tokens (%.1f GB) in %.1f s" % (n_tok, n_tok * 4 / 1e9, time.time() - t0))

    px = PX.Parason(S.CONTIGUOUS_TAGS, group_size=G, **coef)
    out = px.alloc_outputs(n, dev)
    ws = px.alloc_workspace(n, n_tok, dev)
    stream = torch.cuda.current_stream(dev).cuda_stream
    hev = HipEvents()
    ev = [hev.create(), hev.create()]
    c_ev = (ctypes.c_void_p * 2)(ev[0], ev[1])

    def step(timed_scan):
        rc = px.run_timed_raw(tokens.data_ptr(), starts.data_ptr(), lengths.data_ptr(), correct.data_ptr(), n, out,
                              ws.data_ptr(), ws.numel(), stream, c_ev if timed_scan else None)
        if rc != PX.OK:
            raise PX.ParasonError(rc, "parason_run")

    for _ in range(args.warmup):
        step(False)
    torch.cuda.synchronize()

    # whole-step timing
    t0 = time.perf_counter()
    for _ in range(args.steps):
        step(False)
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    ms_per_step = dt * 1e3 / args.steps

    # the dominant kernel, timed with HIP events around its launch
    scan_ms = []
    for _ in range(args.steps):
        step(True)
        scan_ms.append(hev.elapsed_ms(ev[0], ev[1]))
    torch.cuda.synchronize()
    scan_avg = float(np.mean(scan_ms))

    # the measured ceiling: a plain streaming read of the same token buffer,
    # timed the same way on the same stream
    sink = torch.empty(1, dtype=torch.int32, device=dev)
    probe_ms = []
    for i in range(args.warmup + args.steps):
        hev.record(ev[0], stream)
        rc = PX.read_probe_raw(tokens.data_ptr(), 4 * n_tok, sink.data_ptr(), 1, stream)
        if rc != PX.OK:
            raise PX.ParasonError(rc, "parason_read_probe")
        hev.record(ev[1], stream)
        if i >= args.warmup:
            probe_ms.append(hev.elapsed_ms(ev[0], ev[1]))
    torch.cuda.synchronize()
    probe_avg = float(np.mean(probe_ms))

    # sanity of the last step
    fl = out["flags"].cpu().numpy().view(np.uint32)
    n_valid = int(np.sum(fl & PX.FLAG_VALID))
    alg_bytes = 4.0 * n_tok + 44.0 * n
    achieved = alg_bytes / (scan_avg * 1e-3) / 1e9
    traffic = None
    if os.path.exists(PROFILE_TRAFFIC):
        try:
            tr = json.load(open(PROFILE_TRAFFIC))
            if tr.get("workload") == args.workload and tr.get("kernel_source_sha") == kernel_sha():
                traffic = tr.get("bytes_per_launch")
        except Exception:
            traffic = None

    res = {
        "metric": "hot-path throughput (items/s) + achieved % of HBM or MFMA roofline, 1×MI355X",
        "value": n_tok / (ms_per_step * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_per_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int32",
        "data": "synthetic (seeded generator shaped like the paper's rollouts; no dataset or model)",
        "config": {
            "workload": "%s: %d groups x %d rollouts, %d rows, %d tokens (%.1f GB int32)"
                        % (args.workload, n // G, G, n, n_tok, n_tok * 4 / 1e9),
            "rows": n,
            "tokens": n_tok,
            "group_size": G,
            "tag_ids": "contiguous (V-12 .. V-1, V = 151936)",
            "parallelism": "single GPU",
        },
        "rows_per_s": n / (ms_per_step * 1e-3),
        "valid_rows": n_valid,
        "roofline": {
            "kernel": "scan_rows",
            "bound": "hbm",
            "achieved": achieved,
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": achieved / HBM_PEAK_GBS,
            "traffic": traffic,
            "kernel_ms": scan_avg,
            "algorithmic_bytes": alg_bytes,
            "read_ceiling_ms": probe_avg,
            "read_ceiling_gbs": 4.0 * n_tok / (probe_avg * 1e-3) / 1e9,
            "scan_over_ceiling": scan_avg / probe_avg,
            "read_ceiling": "parason_read_probe: plain streaming read of the same token buffer (the scan's "
                            "16-byte nontemporal loads and grid, 8 loads per lane in flight, every 8 KB step "
                            "handed out through a counter in shrinking chunks, no work), timed with HIP events "
                            "on the same stream in the same run",
        },
    }
    if not args.no_cpu_baseline:
        log("timing the CPU oracle on a sample")
        res["cpu_baseline"], ref = cpu_baseline(tokens, starts.cpu().numpy(), lengths.cpu().numpy(),
                                                correct.cpu().numpy(), S.CONTIGUOUS_TAGS, coef, args.cpu_budget)
        res["parity"] = parity_of(out, ref)
        log("parity: %s" % json.dumps(res["parity"]))
    if args.workload == "large" and not args.no_typical_batch:
        # the same step on a batch of the size of one training step (latency-bound, not HBM-bound)
        del tokens, starts, lengths, correct, out, ws
        torch.cuda.empty_cache()
        res["typical_batch"] = time_small_batch("typical", coef, args.steps * 5, args.warmup)
        # and the other small workloads: one group, 32 groups, and 128 groups of log-uniform lengths
        res["small_batches"] = {wl: time_small_batch(wl, coef, args.steps * 10, args.warmup)
                                for wl in ("tiny", "small", "ragged")}
    print(json.dumps(res), flush=True)


GRAPH_CALLS = 8  # accounting calls per captured graph in time_small_batch


def time_small_batch(workload, coef, steps, warmup):
    """Whole-step time of the accounting path on a small batch (wall clock
    around `steps` calls, inputs resident)."""
    import torch

    from paper_2608_24658_amd import parason as PX
    from paper_2608_24658_amd.synth import synth as S

    dev = torch.device("cuda:0")
    G = S.GROUP_SIZE
    P = S.make_params(workload)
    n = S.n_rows_of(workload)
    tokens, starts, lengths, correct = S.device_batch(P, n, device=dev)
    n_tok = int(tokens.numel())
    px = PX.Parason(S.CONTIGUOUS_TAGS, group_size=G, **coef)
    out = px.alloc_outputs(n, dev)
    ws = px.alloc_workspace(n, n_tok, dev)
    stream = torch.cuda.current_stream(dev).cuda_stream

    def step(stream):
        rc = px.run_raw(tokens.data_ptr(), starts.data_ptr(), lengths.data_ptr(), correct.data_ptr(), n, out,
                        ws.data_ptr(), ws.numel(), stream)
        if rc != PX.OK:
            raise PX.ParasonError(rc, "parason_run")

    for _ in range(warmup):
        step(stream)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(steps):
        step(stream)
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / steps
    eager = {k: out[k].clone() for k in ("reward", "flags", "latency", "total")}
    # the same call inside a HIP graph, as in a trainer that captures its whole
    # step (the call allocates nothing and records no memset): GRAPH_CALLS calls
    # captured in one graph and replayed, checked against the eager outputs
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        for _ in range(GRAPH_CALLS):
            step(torch.cuda.current_stream(dev).cuda_stream)
    for _ in range(warmup):
        graph.replay()
    torch.cuda.synchronize()
    reps = max(1, steps // GRAPH_CALLS)
    t0 = time.perf_counter()
    for _ in range(reps):
        graph.replay()
    torch.cuda.synchronize()
    graph_ms = (time.perf_counter() - t0) * 1e3 / (reps * GRAPH_CALLS)
    for k, v in eager.items():
        if not torch.equal(out[k], v):
            raise RuntimeError("graph replay of the %s step differs from the eager step in %s" % (workload, k))
    return {"workload": "%s: %d groups x %d rollouts, %d rows, %d tokens" % (workload, n // G, G, n, n_tok),
            "ms_per_step": ms, "tokens_per_s": n_tok / (ms * 1e-3), "rows_per_s": n / (ms * 1e-3),
            "hip_graph_ms_per_call": graph_ms, "hip_graph_calls_per_replay": GRAPH_CALLS}


def bench_pg(args):
    """The policy-gradient step (advantages + clipped surrogate + gradient) over
    the first half of the large workload's rows: logp, logp_old and the
    gradient for all of its 1.8e10 tokens take 215 GB."""
    import numpy as np
    import torch

    from paper_2608_24658_amd import parason as PX
    from paper_2608_24658_amd.synth import synth as S

    dev = torch.device("cuda:0")
    G = S.GROUP_SIZE
    P = S.make_params(args.workload)
    n_all = S.n_rows_of(args.workload)
    n = n_all // 2 // G * G if args.workload == "large" else n_all
    lengths_h, _ = S.host_rows(P, n)
    starts_h = np.zeros(n, np.int64)
    starts_h[1:] = np.cumsum(lengths_h[:-1].astype(np.int64))
    N = int(lengths_h.astype(np.int64).sum())
    log("pg: %d rows, %d tokens (%.1f GB of logp + logp_old + grad)" % (n, N, 12 * N / 1e9))
    old, new = S.device_logp(P, N, device=dev)
    rng = np.random.default_rng(0)
    reward = torch.as_tensor(rng.choice([-1.0, 1.0, 1.25, 0.8], n).astype(np.float32)).to(dev)
    starts = torch.as_tensor(starts_h).to(dev)
    lengths = torch.as_tensor(lengths_h).to(dev)
    grad = torch.empty_like(new)
    ws = torch.empty(PX.pg_workspace_size(n), dtype=torch.uint8, device=dev)
    for _ in range(args.warmup):
        out = PX.pg_run(reward, new, old, starts, lengths, G, 0.2, 0.28, grad=grad, workspace=ws)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    e0.record()
    for _ in range(args.steps):
        out = PX.pg_run(reward, new, old, starts, lengths, G, 0.2, 0.28, grad=grad, workspace=ws)
    e1.record()
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / args.steps
    ev_ms = e0.elapsed_time(e1) / args.steps
    st = out["stats"].cpu().numpy()
    alg = 12.0 * N + 20.0 * n
    # reference for the same traffic mix: torch's elementwise grad = logp - logp_old
    # (two float streams read, one written; no plan, no reductions)
    for _ in range(2):
        torch.sub(new, old, out=grad)
    torch.cuda.synchronize()
    r0, r1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    r0.record()
    for _ in range(args.steps):
        torch.sub(new, old, out=grad)
    r1.record()
    torch.cuda.synchronize()
    ref_ms = r0.elapsed_time(r1) / args.steps
    res = {
        "metric": "policy-gradient step throughput (tokens/s) + achieved % of HBM roofline, 1×MI355X",
        "value": N / (ms * 1e-3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "fp32",
        "data": "synthetic (seeded log-probabilities; no model)",
        "config": {"workload": "%s, first %d rows: %d tokens" % (args.workload, n, N), "rows": n, "tokens": N,
                   "group_size": G, "clip": [0.2, 0.28]},
        "loss": float(st[0]),
        "clipped": [int(st[2]), int(st[3])],
        "roofline": {"kernel": "pg_run (all launches, HIP events)", "bound": "hbm",
                     "achieved": alg / (ev_ms * 1e-3) / 1e9, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": alg / (ev_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, "traffic": None, "kernel_ms": ev_ms,
                     "algorithmic_bytes": alg},
        "reference": {"what": "torch.sub(logp, logp_old, out=grad): same 12 B per token", "ms": ref_ms,
                      "GB/s": 12.0 * N / (ref_ms * 1e-3) / 1e9},
    }
    print(json.dumps(res), flush=True)


def bench_decode(args):
    """The grammar-constrained decode step on a rollout batch of B sequences
    over the Qwen-size vocabulary (151936 ids, bf16 logits).

    Two regimes, each timed with HIP events over `steps` launches:
      * rollout: the states follow B synthetic rollouts of the typical
        workload token by token (mostly inside text, where only the tag and
        end-of-sequence logits may change);
      * structural: every sequence sits where no text may follow (the first
        step of a rollout: only <think> is allowed), so every row is rewritten
        with -inf: B * V * 2 bytes of HBM writes per launch.  This is the
        kernel's roofline case."""
    import numpy as np
    import torch

    from paper_2608_24658_amd import parason as PX
    from paper_2608_24658_amd.synth import synth as S

    dev = torch.device("cuda:0")
    B, V = args.decode_batch, S.VOCAB
    eos = 151643
    px = PX.Parason(S.CONTIGUOUS_TAGS)
    K = args.steps
    P = S.make_params("typical")
    tok_h, st_h, ln_h, _ = S.host_batch(P, B)
    GRAPH_STEPS = 64
    T = max(args.warmup + K + 1, GRAPH_STEPS)
    assert int(ln_h.min()) >= T, "rollouts shorter than the timed steps"
    idx = st_h[None, :] + np.arange(T, dtype=np.int64)[:, None]
    step_tokens = torch.as_tensor(np.ascontiguousarray(tok_h[idx].astype(np.int32))).to(dev)  # [T, B]
    logits = torch.randn(B, V, device=dev).to(torch.bfloat16)
    states = PX.decode_init(B, dev)

    def timed(fn, n):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for k in range(n):
            fn(k)
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / n

    # rollout regime: the first step masks for <think>, then token k advances every sequence
    px.decode_step(states, logits, None, eos)
    for k in range(args.warmup):
        px.decode_step(states, logits, step_tokens[k], eos)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    roll_ms = timed(lambda k: px.decode_step(states, logits, step_tokens[args.warmup + k], eos), K)
    wall_ms = (time.perf_counter() - t0) * 1e3 / K
    fl = PX.decode_fields(states)[:, 3].cpu().numpy()
    assert not fl.any(), "synthetic rollouts must stay valid"

    # structural regime: fresh states, no token yet: every row but one logit becomes -inf
    fresh = PX.decode_init(B, dev)
    for _ in range(args.warmup):
        px.decode_step(fresh, logits, None, eos)
    struct_ms = timed(lambda k: px.decode_step(fresh, logits, None, eos), K)
    # the first 64 steps of the rollouts as one call sequence (initialisation,
    # the step without a token, 63 steps), eagerly and as a replayed HIP graph
    gstates = torch.empty(B * PX.DECODE_STATE_BYTES, dtype=torch.uint8, device=dev)

    def sequence():
        PX.decode_init(B, dev, states=gstates)
        px.decode_step(gstates, logits, None, eos)
        for k in range(GRAPH_STEPS - 1):
            px.decode_step(gstates, logits, step_tokens[k], eos)

    eager_seq_ms = timed(lambda k: sequence(), 10)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        sequence()
    graph.replay()
    torch.cuda.synchronize()
    graph_seq_ms = timed(lambda k: graph.replay(), 10)
    assert not PX.decode_fields(gstates)[:, 3].any().item(), "synthetic rollouts must stay valid"

    alg = B * (V * 2 + 16 + 16)  # logits written, state read + written
    # reference for a write-only stream of the same size: torch's fill
    for _ in range(args.warmup):
        logits.fill_(float("-inf"))
    fill_ms = timed(lambda k: logits.fill_(float("-inf")), K)
    ach = alg / (struct_ms * 1e-3) / 1e9
    res = {
        "metric": "grammar-constrained decode step: sequences masked per second + % of HBM roofline, 1xMI355X",
        "value": B / (roll_ms * 1e-3),
        "unit": "sequence-steps/s",
        "n_gpus": 1,
        "steps": K,
        "warmup": args.warmup,
        "ms_per_step": roll_ms,
        "wall_ms_per_step": wall_ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (rollout tokens of the typical workload; random logits)",
        "config": {"workload": "decode batch %d, vocab %d, bf16 logits, contiguous tag ids" % (B, V),
                   "batch": B, "vocab": V},
        "structural_ms_per_step": struct_ms,
        "first_64_steps": {"eager_ms_per_step": eager_seq_ms / GRAPH_STEPS,
                           "hip_graph_ms_per_step": graph_seq_ms / GRAPH_STEPS},
        "roofline": {"kernel": "decode_step (structural regime)", "bound": "hbm", "achieved": ach,
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": ach / HBM_PEAK_GBS, "traffic": None,
                     "kernel_ms": struct_ms, "algorithmic_bytes": alg},
        "reference": {"what": "torch fill_ of the same logits (write-only, B * V * 2 bytes)", "ms": fill_ms,
                      "GB/s": B * V * 2 / (fill_ms * 1e-3) / 1e9},
    }
    print(json.dumps(res), flush=True)


def bench_fork(args):
    """Fork/join packing for tool-call execution on a batch of B = 1024
    rollouts of the typical workload, each cut right after one of its
    </Outlines> tags (13.4k-40.2k-token rows, 3-4 entries per outline).

    fork: one context per outline entry (row + <Thread> + the entry's text);
    join: each row followed by its workers' <Thread> ... </Thread> spans (64
    generated tokens each) and </Parallel>.  Timed with HIP events over
    `steps` calls each, outputs pre-sized (no synchronisation inside)."""
    import numpy as np
    import torch

    from paper_2608_24658_amd import parason as PX
    from paper_2608_24658_amd.synth import synth as S

    dev = torch.device("cuda:0")
    B = args.decode_batch
    tags = [int(t) for t in S.CONTIGUOUS_TAGS]
    P = S.make_params("typical")
    tok_h, st_h, ln_h, _ = S.host_batch(P, B)
    end_out = tags[5]
    rng = np.random.default_rng(0)
    cut = np.empty(B, np.int32)
    for i in range(B):
        ends = np.nonzero(tok_h[st_h[i]: st_h[i] + ln_h[i]] == end_out)[0]
        cut[i] = int(rng.choice(ends)) + 1 if len(ends) else ln_h[i]
    tokens = torch.as_tensor(tok_h).to(dev)
    starts = torch.as_tensor(st_h).to(dev)
    lengths = torch.as_tensor(cut).to(dev)
    px = PX.Parason(tags)
    first = px.fork(tokens, starts, lengths, seed=True)  # sizes the outputs
    W, T, _ = (int(x) for x in first["totals"].cpu())
    n_rows_forked = int((first["worker_off"][1:] > first["worker_off"][:-1]).sum().item())

    def timed(fn):
        for _ in range(args.warmup):
            fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(args.steps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / args.steps

    # outputs and workspace allocated once: the timed region holds the C-ABI calls only
    i64, i32 = dict(dtype=torch.int64, device=dev), dict(dtype=torch.int32, device=dev)
    fws = torch.empty(PX._ws_size("parason_fork_workspace_size", B), dtype=torch.uint8, device=dev)
    fo = dict(ctx_tokens=torch.empty(T, **i32), ctx_starts=torch.empty(W, **i64), ctx_lengths=torch.empty(W, **i32),
              ctx_row=torch.empty(W, **i32), ctx_entry=torch.empty(W, **i32), ctx_kind=torch.empty(W, **i32),
              worker_off=torch.empty(B + 1, **i64), row_status=torch.empty(B, **i32), totals=torch.empty(3, **i64))
    f_out = PX.ForkOutputs(W, T, *[fo[k].data_ptr() for k in (
        "ctx_tokens", "ctx_starts", "ctx_lengths", "ctx_row", "ctx_entry", "ctx_kind", "worker_off", "row_status",
        "totals")])
    stream = torch.cuda.current_stream(dev).cuda_stream

    def fork_call():
        rc = px.fork_raw(tokens.data_ptr(), starts.data_ptr(), lengths.data_ptr(), B, PX.FORK_SEED_ENTRY, f_out,
                         fws.data_ptr(), fws.numel(), stream)
        if rc != PX.OK:
            raise PX.ParasonError(rc, "parason_fork")

    fork_ms = timed(fork_call)
    for k, v in fo.items():  # the timed calls wrote what the sizing call did
        if not torch.equal(v, first[k]):
            raise RuntimeError("timed fork calls differ from the first call in %s" % k)
    # workers: their context + 64 generated tokens + </Thread>, packed
    ctx_lens = first["ctx_lengths"].to(torch.int64)
    wlen = ctx_lens + 65
    wstarts = torch.zeros(W, dtype=torch.int64, device=dev)
    wstarts[1:] = torch.cumsum(wlen, 0)[:-1]
    wtokens = torch.full((int(wlen.sum().item()),), 11, dtype=torch.int32, device=dev)
    # copy each context to the front of its worker sequence (setup, not timed)
    idx = torch.repeat_interleave(torch.arange(W, device=dev), ctx_lens)
    within = torch.arange(int(ctx_lens.sum().item()), device=dev) - torch.repeat_interleave(
        first["ctx_starts"], ctx_lens)
    wtokens[wstarts[idx] + within] = first["ctx_tokens"][first["ctx_starts"][idx] + within]
    wtokens[wstarts + wlen - 1] = tags[11]
    wl32 = wlen.to(torch.int32)
    jfirst = px.join(tokens, starts, lengths, first["worker_off"], wtokens, wstarts, wl32)
    JT = int(jfirst["totals"][0].item())
    assert not jfirst["row_status"].any().item()
    jws = torch.empty(PX._ws_size("parason_join_workspace_size", B), dtype=torch.uint8, device=dev)
    jo = dict(tokens=torch.empty(JT, **i32), starts=torch.empty(B + 1, **i64), lengths=torch.empty(B, **i32),
              row_status=torch.empty(B, **i32), totals=torch.empty(2, **i64))
    j_out = PX.JoinOutputs(JT, *[jo[k].data_ptr() for k in ("tokens", "starts", "lengths", "row_status", "totals")])

    def join_call():
        rc = px.join_raw(tokens.data_ptr(), starts.data_ptr(), lengths.data_ptr(), B, first["worker_off"].data_ptr(),
                         wtokens.data_ptr(), wstarts.data_ptr(), wl32.data_ptr(), W, PX.JOIN_CLOSE_PARALLEL, j_out,
                         jws.data_ptr(), jws.numel(), stream)
        if rc != PX.OK:
            raise PX.ParasonError(rc, "parason_join")

    join_ms = timed(join_call)
    for k, v in jo.items():
        if not torch.equal(v, jfirst[k]):
            raise RuntimeError("timed join calls differ from the first call in %s" % k)
    # references at the same sizes: torch's copy_ of T int32 (the contexts' bytes, read and written) and of
    # JT int32 (the joined rows' bytes)
    ref_src = torch.empty(T, dtype=torch.int32, device=dev)
    ref_dst = torch.empty_like(ref_src)
    copy_ms = timed(lambda: ref_dst.copy_(ref_src))
    jcopy_ms = timed(lambda: ref_dst[:JT].copy_(ref_src[:JT]))
    del ref_src, ref_dst
    rows_read = int(cut.astype(np.int64).sum())
    tail = JT - rows_read - B  # each worker's <Thread> ... </Thread> span
    # fork: rows read once, contexts written, 24 B of record per worker, 28 B of offsets/status per row
    fork_bytes = 4 * rows_read + 4 * T + 24 * W + 28 * B
    # join: rows and worker spans read, joined rows written, 36 B per row and 20 B per worker of offsets/checks
    join_bytes = 4 * rows_read + 4 * tail + 4 * JT + 36 * B + 20 * W
    res = {
        "metric": "fork/join packing for tool-call execution: context tokens written per second + % of HBM roofline, "
                  "1xMI355X",
        "value": T / (fork_ms * 1e-3),
        "unit": "context tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": fork_ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int32",
        "data": "synthetic (typical-workload rollouts cut after an outline; generated thread text is filler); outputs "
                "and workspace allocated before the timed calls, whose outputs are checked against the first call's",
        "config": {"workload": "fork %d rows (%d tokens) into %d workers (%d context tokens); join back with 64 "
                               "generated tokens per worker" % (B, rows_read, W, T),
                   "rows": B, "rows_forked": n_rows_forked, "workers": W, "context_tokens": T, "joined_tokens": JT},
        "join_ms": join_ms,
        "join_tokens_per_s": JT / (join_ms * 1e-3),
        "roofline": {"kernel": "parason_fork (all launches, HIP events)", "bound": "hbm",
                     "achieved": fork_bytes / (fork_ms * 1e-3) / 1e9, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": fork_bytes / (fork_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, "traffic": None,
                     "kernel_ms": fork_ms, "algorithmic_bytes": fork_bytes},
        "join_roofline": {"achieved": join_bytes / (join_ms * 1e-3) / 1e9, "unit": "GB/s",
                          "frac": join_bytes / (join_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, "algorithmic_bytes": join_bytes},
        "reference": {"what": "torch copy_ of the context tokens (T int32 read and written, one kernel)",
                      "ms": copy_ms, "GB/s": 8 * T / (copy_ms * 1e-3) / 1e9},
        "join_reference": {"what": "torch copy_ of the joined tokens (JT int32 read and written, one kernel)",
                           "ms": jcopy_ms, "GB/s": 8 * JT / (jcopy_ms * 1e-3) / 1e9},
    }
    print(json.dumps(res), flush=True)


def traffic_summary(d):
    """HBM bytes per scan_rows launch from FETCH_SIZE and WRITE_SIZE (KiB per
    dispatch), each scaled by what the same counter reads for a plain 4 GiB
    device-to-device copy; the algorithmic bytes come from the JSON line the
    profiled FETCH_SIZE run printed."""
    import csv
    import glob

    def per_kernel(sub, counter):
        acc = {}
        for r in csv.DictReader(open(glob.glob(os.path.join(d, sub, "*counter_collection.csv"))[0])):
            if r["Counter_Name"] == counter:
                acc.setdefault(r["Kernel_Name"].split("(")[0].replace("void ", ""), []).append(
                    float(r["Counter_Value"]))
        return {k: sum(v) / len(v) for k, v in acc.items()}, {k: len(v) for k, v in acc.items()}

    cf, _ = per_kernel("prof_copy_fetch", "FETCH_SIZE")
    cw, _ = per_kernel("prof_copy_write", "WRITE_SIZE")
    copy = next(k for k in cf if "copyBuffer" in k)
    fetch_factor = cf[copy] * 1024 / (4 << 30)
    write_factor = cw[copy] * 1024 / (4 << 30)
    f, nf = per_kernel("prof_fetch", "FETCH_SIZE")
    w, _ = per_kernel("prof_write", "WRITE_SIZE")
    scan = next(k for k in f if "scan_rows" in k)
    line = [ln for ln in open(os.path.join(d, "prof_fetch.log")) if ln.startswith("{")][-1]
    run = json.loads(line)
    alg = run["roofline"]["algorithmic_bytes"]
    traffic = f[scan] * 1024 / fetch_factor + w[scan] * 1024 / write_factor
    rec = {"kernel": "scan_rows", "workload": run["config"]["workload"].split(":")[0],
           "kernel_source_sha": kernel_sha(), "fetch_kib_per_launch": f[scan], "write_kib_per_launch": w[scan],
           "launches": nf[scan],
           "copy_calibration": {"kernel": copy, "bytes_read": 4 << 30, "bytes_written": 4 << 30,
                                "fetch_kib": cf[copy], "write_kib": cw[copy], "fetch_factor": fetch_factor,
                                "write_factor": write_factor},
           "bytes_per_launch": traffic, "algorithmic_bytes_per_launch": alg,
           "traffic_over_algorithmic": traffic / alg,
           "other_kernels_gb_per_launch": {k: [f[k] * 1024 / fetch_factor / 1e9, w.get(k, 0.0) * 1024 / write_factor / 1e9]
                                           for k in f if k.startswith("pk::") or "pk::" in k}}
    # a second calibration point of known size from the same FETCH_SIZE run: the
    # read probe reads each of the run's tokens exactly once (4 B per token)
    probe = next((k for k in f if "read_probe" in k), None)
    if probe is not None:
        probe_bytes = 4.0 * run["config"]["tokens"]
        rec["probe_check"] = {"kernel": probe, "bytes_read": probe_bytes, "fetch_kib": f[probe],
                              "fetch_factor": f[probe] * 1024 / probe_bytes,
                              "calibrated_over_read": f[probe] * 1024 / fetch_factor / probe_bytes}
    with open(PROFILE_TRAFFIC, "w") as fh:
        json.dump(rec, fh, indent=1)
    print(json.dumps(rec, indent=1))


def kernel_sha():
    """Hash of the sources of the accounting path's kernels and launches, with
    comments and whitespace removed (the other entry points of the library live
    in files of their own and do not enter it)."""
    import hashlib
    import re

    h = hashlib.sha256()
    for p in ("paper_2608_24658_amd/csrc/device_common.h", "paper_2608_24658_amd/csrc/parason_kernels.h",
              "paper_2608_24658_amd/csrc/abi_common.h", "paper_2608_24658_amd/csrc/parason.hip"):
        src = open(os.path.join(ROOT, p)).read()
        src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
        src = re.sub(r"//[^\n]*", "", src)
        h.update(re.sub(r"\s+", "", src).encode())
    return h.hexdigest()[:16]


if __name__ == "__main__":
    main()
