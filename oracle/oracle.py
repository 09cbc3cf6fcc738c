"""ctypes binding of the CPU oracle (``parason_oracle.c``).

TEST INFRASTRUCTURE.  Only the tests, the smoke check and the CPU-baseline leg
of the benchmark may import this module; the product path never does.

The oracle is plain single-threaded C: a recursive-descent parser with one
function per production of the grammar in the figure "Context-Free Grammar for
Parason" (Sec. 3.2), the latency of Sec. 4 ("Evaluation"), the branch-token
ratios and eta of Sec. 3.3, and the reward of Definition 3.1 (Sec. 3.3) in IEEE
double precision.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "parason_oracle.c")
LIB = os.path.join(HERE, "liboracle.so")

# Field order of oracle_row_t.
ROW_DTYPE = np.dtype(
    [
        ("total", np.int32),
        ("latency", np.int32),
        ("n_subtask", np.int32),
        ("n_trial", np.int32),
        ("n_blocks", np.int32),
        ("max_depth", np.int32),
        ("first_error_pos", np.int32),
        ("flags", np.uint32),
    ]
)

F_VALID = 1 << 0
F_TRUNCATED = 1 << 1
F_COUNT_MISMATCH = 1 << 2
F_TRIGGERED = 1 << 3

CFG_INVALID_KEEPS_CORRECTNESS = 1 << 0
CFG_BATCH_STATS = 1 << 1
CFG_LENIENT_GAPS = 1 << 3  # Text runs allowed between the structural tags of a parallel region

METRICS = (
    "rows", "valid", "triggered", "correct", "truncated", "count_mismatch",
    "sum_total", "sum_latency", "sum_subtask", "sum_trial",
    "trigger_ratio", "acceleration", "mean_latency", "mean_total", "mean_saved",
    "subtask_share", "trial_share", "accuracy", "mean_reward",
)

TAG_NAMES = (
    "<think>", "</think>", "<Parallel>", "</Parallel>", "<Outlines>", "</Outlines>",
    "<Subtask>", "</Subtask>", "<Trial>", "</Trial>", "<Thread>", "</Thread>",
)

_lib = None


def build(force: bool = False) -> str:
    """Compile the oracle with gcc (no fast-math, no FMA contraction)."""
    if force or not os.path.exists(LIB) or os.path.getmtime(LIB) < os.path.getmtime(SRC):
        tmp = LIB + ".tmp%d" % os.getpid()
        cmd = [
            "gcc", "-O2", "-std=c99", "-fPIC", "-shared", "-ffp-contract=off",
            "-fno-fast-math", "-Wall", "-Wextra", "-o", tmp, SRC, "-lm", "-lpthread",
        ]
        subprocess.check_call(cmd)
        os.replace(tmp, LIB)
    return LIB


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB):
            build()
        L = ctypes.CDLL(LIB)
        L.oracle_eval_rows.restype = ctypes.c_int
        L.oracle_eval_rows.argtypes = [
            ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64,
            ctypes.c_void_p, ctypes.c_uint32, ctypes.c_void_p,
        ]
        L.oracle_group_reward.restype = ctypes.c_int
        L.oracle_group_reward.argtypes = [
            ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32,
            ctypes.c_void_p, ctypes.c_uint32, ctypes.c_void_p, ctypes.c_void_p,
            ctypes.c_void_p, ctypes.c_void_p,
        ]
        L.oracle_batch_metrics.restype = ctypes.c_int
        L.oracle_batch_metrics.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64,
                                           ctypes.c_void_p]
        _lib = L
    return _lib


def _ptr(a: np.ndarray) -> int:
    return a.ctypes.data


def eval_rows(tokens, starts, lengths, tag_ids, cfg_flags: int = 0) -> np.ndarray:
    """Per-row accounting.  Row i is tokens[starts[i] : starts[i] + lengths[i]].
    cfg_flags: CFG_LENIENT_GAPS or 0."""
    tokens = np.ascontiguousarray(tokens, dtype=np.int32)
    starts = np.ascontiguousarray(starts, dtype=np.int64)
    lengths = np.ascontiguousarray(lengths, dtype=np.int32)
    tag_ids = np.ascontiguousarray(tag_ids, dtype=np.int32)
    assert tag_ids.shape == (12,)
    n = starts.shape[0]
    assert lengths.shape == (n,)
    if n and tokens.size:
        assert starts.min() >= 0 and (starts + lengths).max() <= tokens.size
    out = np.zeros(n, dtype=ROW_DTYPE)
    if n == 0:
        return out
    if tokens.size == 0:
        tokens = np.zeros(1, dtype=np.int32)
    rc = lib().oracle_eval_rows(_ptr(tokens), _ptr(starts), _ptr(lengths), n, _ptr(tag_ids),
                                cfg_flags & CFG_LENIENT_GAPS, _ptr(out))
    if rc != 0:
        raise RuntimeError("oracle_eval_rows failed: %d" % rc)
    return out


def eval_stream(stream, tag_ids, cfg_flags: int = 0) -> np.void:
    """Accounting of a single token stream."""
    s = np.asarray(stream, dtype=np.int32)
    return eval_rows(s, np.array([0]), np.array([s.size]), tag_ids, cfg_flags)[0]


def group_reward(rows: np.ndarray, correct, group_size: int, alpha: float, beta_subtask: float,
                 beta_trial: float, rho: float, rho_clip: float, cfg_flags: int = 0):
    """Reward of Definition 3.1 per row, plus R_subtask, R_trial and eta (all float64).

    With CFG_BATCH_STATS in cfg_flags, mu and sigma are taken over the whole
    batch (the batch is one normalisation group) instead of each G rows."""
    if cfg_flags & CFG_BATCH_STATS:
        group_size = len(rows)
        if group_size == 0:
            z = np.zeros(0)
            return z, z, z, z
    rows = np.ascontiguousarray(rows, dtype=ROW_DTYPE)
    correct = np.ascontiguousarray(correct, dtype=np.uint8)
    n = rows.shape[0]
    params = np.array([alpha, beta_subtask, beta_trial, rho, rho_clip], dtype=np.float64)
    reward = np.zeros(n, np.float64)
    r_sub = np.zeros(n, np.float64)
    r_tri = np.zeros(n, np.float64)
    eta = np.zeros(n, np.float64)
    if n == 0:
        return reward, r_sub, r_tri, eta
    rc = lib().oracle_group_reward(
        _ptr(rows), _ptr(correct), n, group_size, _ptr(params), cfg_flags,
        _ptr(reward), _ptr(r_sub), _ptr(r_tri), _ptr(eta),
    )
    if rc != 0:
        raise ValueError("oracle_group_reward failed: %d (n_rows %% group_size must be 0)" % rc)
    return reward, r_sub, r_tri, eta


def row_acceleration(rows: np.ndarray):
    """Per-row acceleration ratio and saved tokens (float64, int64).

    Acceleration = total tokens / longest-path tokens (Table 4 caption;
    Table 5 divides generated by latency tokens), 1 for an empty row; saved
    tokens = generated - latency (Table 5)."""
    total = rows["total"].astype(np.int64)
    lat = rows["latency"].astype(np.int64)
    accel = np.ones(len(rows), np.float64)
    nz = total > 0
    accel[nz] = total[nz].astype(np.float64) / lat[nz].astype(np.float64)
    return accel, total - lat


def batch_metrics(rows: np.ndarray, correct, reward) -> dict:
    """Batch metrics of Tables 2, 4 and 5 (see oracle_batch_metrics)."""
    rows = np.ascontiguousarray(rows, dtype=ROW_DTYPE)
    correct = np.ascontiguousarray(correct, dtype=np.uint8)
    reward = np.ascontiguousarray(reward, dtype=np.float64)
    m = np.zeros(len(METRICS), np.float64)
    n = rows.shape[0]
    if n == 0:
        rows = np.zeros(1, dtype=ROW_DTYPE)
        correct = np.zeros(1, np.uint8)
        reward = np.zeros(1)
    rc = lib().oracle_batch_metrics(_ptr(rows), _ptr(correct), _ptr(reward), n, _ptr(m))
    assert rc == 0
    return dict(zip(METRICS, m.tolist()))
