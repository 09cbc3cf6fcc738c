"""Seeded synthetic reasoning trajectories shaped like the paper's workloads.

Input generation only.  The paper's rollouts (its own model on AIME24/25,
Math500 and AMC) are not available; these streams stand in for them.  Shapes
come from the paper's reported statistics:

* groups of G = 8 rollouts per prompt (Sec. 4, "Training Framework");
* 90% of rows contain at least one <Parallel> block (trigger ratios of
  53.7-98.8%, Table 4); 1-3 top-level blocks;
* a block is Trial with probability 0.655 (the Trial share of parallelizable
  steps for DeepSeek-V4 on HLE, Table 1), Subtask otherwise; one type per block
  (Sec. 3.2); Trial blocks have 1-4 entries, Subtask blocks 2-4, and a Subtask
  thread holds a nested Trial block with probability 0.5 (the structure of
  Figure 3);
* span weights chosen so that total / latency is close to the reported 1.7x
  (abstract; Tables 4 and 5);
* correct with probability 0.8 (average accuracy about 78-80%, Table 4).

Token ids: vocabulary of V = 151,936 ids (an assumption: the size of the
Qwen3-family vocabulary; the paper does not state it) with the 12 tags at the
top, V-12 .. V-1, in the order of the tag_ids argument.  Text ids are uniform
over the other ids.

The five workloads (G = 8; "batch" = prompts):

======  ===========================================================  ====
name    rows and lengths                                              seed
======  ===========================================================  ====
tiny    1 group; total uniform in [2000, 5000] (latency about 2k, the   0
        smallest budget of Table 3)
small   32 groups, lengths as tiny                                      1
typical 256 groups; total uniform in [13400, 40200] (mean 26.8k:        2
        latency 15.7k at 1.71x, Table 4); 1% of thread bodies x100
large   89,000 groups; total uniform in [25150, 75450] (mean 50.3k,     3
        the hard rows of Table 5); about 3.6e10 tokens, 143 GB
ragged  128 groups; total log-uniform over [1, 50300]               4
        (P(L) ~ 1/L); 5% of rows truncated at a uniform position
======  ===========================================================  ====
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
DEV_LIB = os.path.join(HERE, "libparason_synth.so")
HOST_LIB = os.path.join(HERE, "libparason_synth_host.so")

VOCAB = 151936
GROUP_SIZE = 8
CONTIGUOUS_TAGS = np.arange(VOCAB - 12, VOCAB, dtype=np.int32)
# A scattered set of tag ids (used by tests of the general tag matcher).
SCATTERED_TAGS = np.array([151930, 17, 90001, 5, 65535, 65536, 1, 140000, 777, 31337, 100000, 2], dtype=np.int32)


class SynthParams(ctypes.Structure):
    _fields_ = [
        ("seed_lo", ctypes.c_uint32),
        ("seed_hi", ctypes.c_uint32),
        ("vocab", ctypes.c_int32),
        ("tag_ids", ctypes.c_int32 * 12),
        ("sorted_tags", ctypes.c_int32 * 12),
        ("len_kind", ctypes.c_int32),
        ("len_lo", ctypes.c_int32),
        ("len_hi", ctypes.c_int32),
        ("p_trigger", ctypes.c_uint32),
        ("p_trial", ctypes.c_uint32),
        ("p_nest", ctypes.c_uint32),
        ("p_outlier", ctypes.c_uint32),
        ("p_trunc", ctypes.c_uint32),
        ("p_correct", ctypes.c_uint32),
        ("w_main", ctypes.c_uint32),
        ("w_entry", ctypes.c_uint32),
        ("w_body", ctypes.c_uint32),
        ("w_answer", ctypes.c_uint32),
        ("outlier_mult", ctypes.c_int32),
        ("max_blocks", ctypes.c_int32),
    ]


def _p(x: float) -> int:
    return min(int(round(x * 2.0 ** 32)), 2 ** 32 - 1)


WORKLOADS = {
    "tiny": dict(groups=1, seed=0, len_kind=0, len_lo=2000, len_hi=5000),
    "small": dict(groups=32, seed=1, len_kind=0, len_lo=2000, len_hi=5000),
    "typical": dict(groups=256, seed=2, len_kind=0, len_lo=13400, len_hi=40200, p_outlier=0.01),
    "large": dict(groups=89000, seed=3, len_kind=0, len_lo=25150, len_hi=75450),
    "ragged": dict(groups=128, seed=4, len_kind=1, len_lo=1, len_hi=50300, p_trunc=0.05),
}


def make_params(workload: str | dict = "tiny", tag_ids=None, seed=None, **over) -> SynthParams:
    w = dict(WORKLOADS[workload]) if isinstance(workload, str) else dict(workload)
    w.update(over)
    tags = np.asarray(CONTIGUOUS_TAGS if tag_ids is None else tag_ids, dtype=np.int32)
    assert tags.shape == (12,) and len(set(tags.tolist())) == 12
    P = SynthParams()
    s = int(w["seed"] if seed is None else seed)
    P.seed_lo, P.seed_hi = s & 0xFFFFFFFF, (s >> 32) & 0xFFFFFFFF
    P.vocab = int(w.get("vocab", VOCAB))
    assert tags.min() >= 0 and tags.max() < P.vocab
    for i in range(12):
        P.tag_ids[i] = int(tags[i])
    for i, t in enumerate(sorted(tags.tolist())):
        P.sorted_tags[i] = int(t)
    P.len_kind = int(w["len_kind"])
    P.len_lo, P.len_hi = int(w["len_lo"]), int(w["len_hi"])
    P.p_trigger = _p(w.get("p_trigger", 0.9))
    P.p_trial = _p(w.get("p_trial", 0.655))
    P.p_nest = _p(w.get("p_nest", 0.5))
    P.p_outlier = _p(w.get("p_outlier", 0.0))
    P.p_trunc = _p(w.get("p_trunc", 0.0))
    P.p_correct = _p(w.get("p_correct", 0.8))
    P.w_main = int(w.get("w_main", 400))
    P.w_entry = int(w.get("w_entry", 40))
    P.w_body = int(w.get("w_body", 1400))
    P.w_answer = int(w.get("w_answer", 100))
    P.outlier_mult = int(w.get("outlier_mult", 100))
    P.max_blocks = int(w.get("max_blocks", 3))
    return P


def n_rows_of(workload: str) -> int:
    return WORKLOADS[workload]["groups"] * GROUP_SIZE


_host = None
_dev = None


def host_lib():
    global _host
    if _host is None:
        if not os.path.exists(HOST_LIB):
            raise RuntimeError("generator host library not built: run __graft_entry__.build()")
        L = ctypes.CDLL(HOST_LIB)
        L.synth_rows_host.restype = ctypes.c_int
        L.synth_rows_host.argtypes = [ctypes.POINTER(SynthParams), ctypes.c_uint64, ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p]
        L.synth_row_tokens_host.restype = ctypes.c_int64
        L.synth_row_tokens_host.argtypes = [ctypes.POINTER(SynthParams), ctypes.c_uint64, ctypes.c_uint64, ctypes.c_void_p, ctypes.c_int64]
        L.synth_logp_host.restype = ctypes.c_int
        L.synth_logp_host.argtypes = [ctypes.POINTER(SynthParams), ctypes.c_uint64, ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p]
        _host = L
    return _host


def dev_lib():
    global _dev
    if _dev is None:
        if not os.path.exists(DEV_LIB):
            raise RuntimeError("generator device library not built: run __graft_entry__.build()")
        L = ctypes.CDLL(DEV_LIB)
        for f in ("synth_rows_device", "synth_text_device", "synth_tags_device", "synth_logp_device"):
            getattr(L, f).restype = ctypes.c_int
        L.synth_rows_device.argtypes = [ctypes.POINTER(SynthParams), ctypes.c_uint64, ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
        L.synth_text_device.argtypes = [ctypes.POINTER(SynthParams), ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p]
        L.synth_tags_device.argtypes = [ctypes.POINTER(SynthParams), ctypes.c_uint64, ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p]
        L.synth_logp_device.argtypes = [ctypes.POINTER(SynthParams), ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p]
        _dev = L
    return _dev


def host_rows(P: SynthParams, n_rows: int, row0: int = 0):
    """Lengths and correctness bits of rows row0 .. row0+n_rows (host mirror)."""
    lengths = np.zeros(n_rows, np.int32)
    correct = np.zeros(n_rows, np.uint8)
    rc = host_lib().synth_rows_host(ctypes.byref(P), row0, n_rows, lengths.ctypes.data, correct.ctypes.data)
    assert rc == 0
    return lengths, correct


def host_row_tokens(P: SynthParams, row: int, flat0: int, length: int) -> np.ndarray:
    """Tokens of one row whose first token sits at flat index flat0 of the batch."""
    out = np.zeros(max(length, 1), np.int32)
    n = host_lib().synth_row_tokens_host(ctypes.byref(P), row, flat0, out.ctypes.data, out.size)
    assert n == length, (n, length)
    return out[:length]


def host_batch(P: SynthParams, n_rows: int):
    """A whole packed batch on the host: (tokens, starts, lengths, correct)."""
    lengths, correct = host_rows(P, n_rows)
    starts = np.zeros(n_rows, np.int64)
    if n_rows:
        starts[1:] = np.cumsum(lengths[:-1].astype(np.int64))
    total = int(lengths.astype(np.int64).sum())
    tokens = np.zeros(max(total, 4), np.int32)
    for i in range(n_rows):
        if lengths[i]:
            tokens[starts[i]: starts[i] + lengths[i]] = host_row_tokens(P, i, int(starts[i]), int(lengths[i]))
    return tokens[:total] if total else tokens[:0], starts, lengths, correct


def device_batch(P: SynthParams, n_rows: int, device="cuda", pad: int = 0):
    """A whole packed batch generated on the GPU (torch tensors on `device`).

    Returns (tokens, starts, lengths, correct).  `pad` extra int32 slots follow
    the last row (filled with Text ids)."""
    import torch

    L = dev_lib()
    stream = torch.cuda.current_stream(device).cuda_stream
    lengths = torch.empty(n_rows, dtype=torch.int32, device=device)
    correct = torch.empty(n_rows, dtype=torch.uint8, device=device)
    if n_rows:
        rc = L.synth_rows_device(ctypes.byref(P), 0, n_rows, lengths.data_ptr(), correct.data_ptr(), stream)
        assert rc == 0, rc
    starts = torch.zeros(n_rows, dtype=torch.int64, device=device)
    if n_rows > 1:
        torch.cumsum(lengths[:-1].to(torch.int64), 0, out=starts[1:])
    total = int(lengths.to(torch.int64).sum().item()) if n_rows else 0
    tokens = torch.empty(total + pad, dtype=torch.int32, device=device)
    if total + pad:
        rc = L.synth_text_device(ctypes.byref(P), tokens.data_ptr(), total + pad, stream)
        assert rc == 0, rc
    if n_rows:
        rc = L.synth_tags_device(ctypes.byref(P), 0, n_rows, starts.data_ptr(), tokens.data_ptr(), stream)
        assert rc == 0, rc
    return tokens, starts, lengths, correct


def host_logp(P: SynthParams, p0: int, n: int):
    """(logp_old, logp) float32 for flat positions [p0, p0 + n) (host mirror)."""
    old = np.zeros(max(n, 1), np.float32)
    new = np.zeros(max(n, 1), np.float32)
    rc = host_lib().synth_logp_host(ctypes.byref(P), p0, n, old.ctypes.data, new.ctypes.data)
    assert rc == 0
    return old[:n], new[:n]


def device_logp(P: SynthParams, n: int, device="cuda"):
    """(logp_old, logp) float32 device tensors of n positions."""
    import torch

    old = torch.empty(n, dtype=torch.float32, device=device)
    new = torch.empty(n, dtype=torch.float32, device=device)
    if n:
        rc = dev_lib().synth_logp_device(ctypes.byref(P), old.data_ptr(), new.data_ptr(), n,
                                         torch.cuda.current_stream(device).cuda_stream)
        assert rc == 0, rc
    return old, new
