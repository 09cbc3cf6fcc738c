"""Python binding of libparason.so (argument marshalling only).

Every step of the path runs in the HIP kernels behind the C-ABI declared in
``include/parason.h``; this module turns torch tensors into device pointers and
passes torch's current HIP stream.  It raises if the library is missing: there
is no fallback.
"""
from __future__ import annotations

import ctypes
import os

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libparason.so")

OK = 0
ERR_NULL, ERR_SIZE, ERR_GROUP, ERR_WORKSPACE, ERR_TAGS, ERR_PARAM, ERR_ALIGN, ERR_HIP, ERR_DEVICE, ERR_SCRATCH = \
    range(-1, -11, -1)
NOALLOC_SCRATCH_BYTES = 128 << 20

FLAG_VALID = 1 << 0
FLAG_TRUNCATED = 1 << 1
FLAG_COUNT_MISMATCH = 1 << 2
FLAG_TRIGGERED = 1 << 3
FLAG_DEPTH_LIMIT = 1 << 8
FLAG_WS_OVERFLOW = 1 << 9
FLAG_BAD_ROW = 1 << 10

CFG_INVALID_KEEPS_CORRECTNESS = 1 << 0
CFG_BATCH_STATS = 1 << 1
CFG_TAG_COMPARE = 1 << 2
CFG_LENIENT_GAPS = 1 << 3

METRICS = (
    "rows", "valid", "triggered", "correct", "truncated", "count_mismatch",
    "sum_total", "sum_latency", "sum_subtask", "sum_trial",
    "trigger_ratio", "acceleration", "mean_latency", "mean_total", "mean_saved",
    "subtask_share", "trial_share", "accuracy", "mean_reward",
)

MAX_DEPTH = 1 << 20
MAX_OPEN_ENTRIES = 1 << 24

EXPORTED = ("parason_create", "parason_workspace_size", "parason_run", "parason_run_timed", "parason_destroy",
            "parason_strerror", "parason_pg_workspace_size", "parason_pg_run", "parason_decode_init",
            "parason_decode_step", "parason_fork_workspace_size", "parason_join_workspace_size", "parason_fork",
            "parason_join", "parason_read_probe", "parason_run_noalloc")

FORK_SEED_ENTRY = 1 << 0
JOIN_CLOSE_PARALLEL = 1 << 0
JOIN_APPEND_ONLY = 1 << 1
PACK_NO_OUTLINE_END = 1 << 0
PACK_NO_OUTLINE = 1 << 1
PACK_BAD_ENTRY = 1 << 2
PACK_BAD_THREAD = 1 << 3
PACK_TOO_LONG = 1 << 4
PACK_BAD_ROW = 1 << 5

DECODE_ERROR = 1 << 0
DECODE_DONE = 1 << 1
DTYPE_F32, DTYPE_BF16, DTYPE_F16 = 0, 1, 2
DECODE_STATE_BYTES = 16

PG_STATS = ("loss", "tokens", "clip_high", "clip_low")


class Config(ctypes.Structure):
    _fields_ = [
        ("tag_ids", ctypes.c_int32 * 12),
        ("group_size", ctypes.c_int32),
        ("alpha", ctypes.c_double),
        ("beta_subtask", ctypes.c_double),
        ("beta_trial", ctypes.c_double),
        ("rho", ctypes.c_double),
        ("rho_clip", ctypes.c_double),
        ("flags", ctypes.c_uint32),
    ]


class PgConfig(ctypes.Structure):
    _fields_ = [("group_size", ctypes.c_int32), ("clip_low", ctypes.c_double), ("clip_high", ctypes.c_double)]


class Outputs(ctypes.Structure):
    _fields_ = [
        ("total", ctypes.c_void_p),
        ("latency", ctypes.c_void_p),
        ("n_subtask", ctypes.c_void_p),
        ("n_trial", ctypes.c_void_p),
        ("n_blocks", ctypes.c_void_p),
        ("max_depth", ctypes.c_void_p),
        ("first_error_pos", ctypes.c_void_p),
        ("flags", ctypes.c_void_p),
        ("reward", ctypes.c_void_p),
        ("r_subtask", ctypes.c_void_p),
        ("r_trial", ctypes.c_void_p),
        ("eta", ctypes.c_void_p),
        ("metrics", ctypes.c_void_p),
        ("accel", ctypes.c_void_p),
        ("saved", ctypes.c_void_p),
    ]


class ForkOutputs(ctypes.Structure):
    _fields_ = [
        ("max_workers", ctypes.c_int64),
        ("ctx_capacity", ctypes.c_int64),
        ("ctx_tokens", ctypes.c_void_p),
        ("ctx_starts", ctypes.c_void_p),
        ("ctx_lengths", ctypes.c_void_p),
        ("ctx_row", ctypes.c_void_p),
        ("ctx_entry", ctypes.c_void_p),
        ("ctx_kind", ctypes.c_void_p),
        ("worker_off", ctypes.c_void_p),
        ("row_status", ctypes.c_void_p),
        ("totals", ctypes.c_void_p),
    ]


class JoinOutputs(ctypes.Structure):
    _fields_ = [
        ("capacity", ctypes.c_int64),
        ("tokens", ctypes.c_void_p),
        ("starts", ctypes.c_void_p),
        ("lengths", ctypes.c_void_p),
        ("row_status", ctypes.c_void_p),
        ("totals", ctypes.c_void_p),
    ]


INT_FIELDS = ("total", "latency", "n_subtask", "n_trial", "n_blocks", "max_depth", "first_error_pos")
FLOAT_FIELDS = ("reward", "r_subtask", "r_trial", "eta", "accel")
OPTIONAL_FIELDS = ("r_subtask", "r_trial", "eta", "metrics", "accel", "saved")

_lib = None


class ParasonError(RuntimeError):
    def __init__(self, status: int, what: str):
        self.status = status
        super().__init__("%s failed: %s (%d)" % (what, strerror(status), status))


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(
                "libparason.so is not built (%s); run __graft_entry__.build() -- there is no fallback" % LIB_PATH)
        L = ctypes.CDLL(LIB_PATH)
        L.parason_create.restype = ctypes.c_int
        L.parason_create.argtypes = [ctypes.POINTER(Config), ctypes.POINTER(ctypes.c_void_p)]
        L.parason_workspace_size.restype = ctypes.c_int
        L.parason_workspace_size.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64, ctypes.POINTER(ctypes.c_size_t)]
        L.parason_run.restype = ctypes.c_int
        L.parason_run.argtypes = [
            ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64,
            ctypes.POINTER(Outputs), ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p,
        ]
        L.parason_run_noalloc.restype = ctypes.c_int
        L.parason_run_noalloc.argtypes = [
            ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64,
            ctypes.c_int64, ctypes.POINTER(Outputs), ctypes.c_void_p,
        ]
        L.parason_run_timed.restype = ctypes.c_int
        L.parason_run_timed.argtypes = L.parason_run.argtypes + [ctypes.c_void_p]
        L.parason_destroy.restype = None
        L.parason_destroy.argtypes = [ctypes.c_void_p]
        L.parason_pg_workspace_size.restype = ctypes.c_int
        L.parason_pg_workspace_size.argtypes = [ctypes.c_int64, ctypes.POINTER(ctypes.c_size_t)]
        L.parason_pg_run.restype = ctypes.c_int
        L.parason_pg_run.argtypes = [
            ctypes.POINTER(PgConfig), ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
            ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
            ctypes.c_size_t, ctypes.c_void_p,
        ]
        L.parason_decode_init.restype = ctypes.c_int
        L.parason_decode_init.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p]
        L.parason_decode_step.restype = ctypes.c_int
        L.parason_decode_step.argtypes = [
            ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p, ctypes.c_int64,
            ctypes.c_int64, ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p,
        ]
        for name in ("parason_fork_workspace_size", "parason_join_workspace_size"):
            getattr(L, name).restype = ctypes.c_int
            getattr(L, name).argtypes = [ctypes.c_int64, ctypes.POINTER(ctypes.c_size_t)]
        L.parason_fork.restype = ctypes.c_int
        L.parason_fork.argtypes = [
            ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64, ctypes.c_uint32,
            ctypes.POINTER(ForkOutputs), ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p,
        ]
        L.parason_join.restype = ctypes.c_int
        L.parason_join.argtypes = [
            ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64, ctypes.c_void_p,
            ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64, ctypes.c_uint32,
            ctypes.POINTER(JoinOutputs), ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p,
        ]
        L.parason_read_probe.restype = ctypes.c_int
        L.parason_read_probe.argtypes = [ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p, ctypes.c_int64,
                                         ctypes.c_void_p]
        L.parason_strerror.restype = ctypes.c_char_p
        L.parason_strerror.argtypes = [ctypes.c_int]
        _lib = L
    return _lib


def strerror(status: int) -> str:
    return lib().parason_strerror(status).decode()


def make_config(tag_ids, group_size=8, alpha=0.1, beta_subtask=0.0, beta_trial=0.1, rho=0.5, rho_clip=0.25,
                flags=0) -> Config:
    c = Config()
    ids = [int(t) for t in tag_ids]
    if len(ids) != 12:
        raise ValueError("tag_ids must have 12 entries")
    for i, t in enumerate(ids):
        c.tag_ids[i] = t
    c.group_size = int(group_size)
    c.alpha, c.beta_subtask, c.beta_trial = float(alpha), float(beta_subtask), float(beta_trial)
    c.rho, c.rho_clip = float(rho), float(rho_clip)
    c.flags = int(flags)
    return c


class Parason:
    """Handle of the C-ABI (immutable configuration)."""

    def __init__(self, tag_ids, group_size=8, alpha=0.1, beta_subtask=0.0, beta_trial=0.1, rho=0.5,
                 rho_clip=0.25, flags=0):
        self.config = make_config(tag_ids, group_size, alpha, beta_subtask, beta_trial, rho, rho_clip, flags)
        h = ctypes.c_void_p()
        rc = lib().parason_create(ctypes.byref(self.config), ctypes.byref(h))
        if rc != OK:
            raise ParasonError(rc, "parason_create")
        self._h = h

    @property
    def group_size(self) -> int:
        return self.config.group_size

    def close(self):
        if getattr(self, "_h", None):
            lib().parason_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def workspace_size(self, n_traj: int, total_tokens: int) -> int:
        b = ctypes.c_size_t()
        rc = lib().parason_workspace_size(self._h, int(n_traj), int(total_tokens), ctypes.byref(b))
        if rc != OK:
            raise ParasonError(rc, "parason_workspace_size")
        return b.value

    def alloc_outputs(self, n_traj: int, device, derived: bool = True, metrics: bool = False) -> dict:
        import torch

        out = {k: torch.empty(n_traj, dtype=torch.int32, device=device) for k in INT_FIELDS}
        out["flags"] = torch.empty(n_traj, dtype=torch.int32, device=device)  # uint32 bits
        out["reward"] = torch.empty(n_traj, dtype=torch.float32, device=device)
        if derived:
            for k in ("r_subtask", "r_trial", "eta", "accel"):
                out[k] = torch.empty(n_traj, dtype=torch.float32, device=device)
            out["saved"] = torch.empty(n_traj, dtype=torch.int32, device=device)
        if metrics:
            out["metrics"] = torch.empty(len(METRICS), dtype=torch.float64, device=device)
        return out

    def alloc_workspace(self, n_traj: int, total_tokens: int, device):
        import torch

        return torch.empty(self.workspace_size(n_traj, total_tokens), dtype=torch.uint8, device=device)

    def run_raw(self, tokens_ptr, starts_ptr, lengths_ptr, correct_ptr, n_traj, out: dict, ws_ptr, ws_bytes,
                stream) -> int:
        """Direct C-ABI call with raw device pointers; returns the status."""
        o = Outputs()
        for k in INT_FIELDS + ("flags", "reward"):
            setattr(o, k, out[k].data_ptr())
        for k in OPTIONAL_FIELDS:
            setattr(o, k, out[k].data_ptr() if k in out and out[k] is not None else None)
        return lib().parason_run(self._h, tokens_ptr, starts_ptr, lengths_ptr, correct_ptr, int(n_traj),
                                 ctypes.byref(o), ws_ptr, int(ws_bytes), stream)

    def run_noalloc_raw(self, tokens_ptr, starts_ptr, lengths_ptr, correct_ptr, n_traj, total_tokens, out: dict,
                        stream) -> int:
        """parason_run_noalloc (no workspace: the library's static scratch); returns the status."""
        o = Outputs()
        for k in INT_FIELDS + ("flags", "reward"):
            setattr(o, k, out[k].data_ptr())
        for k in OPTIONAL_FIELDS:
            setattr(o, k, out[k].data_ptr() if k in out and out[k] is not None else None)
        return lib().parason_run_noalloc(self._h, tokens_ptr, starts_ptr, lengths_ptr, correct_ptr, int(n_traj),
                                         int(total_tokens), ctypes.byref(o), stream)

    def run_timed_raw(self, tokens_ptr, starts_ptr, lengths_ptr, correct_ptr, n_traj, out: dict, ws_ptr, ws_bytes,
                      stream, scan_events) -> int:
        """parason_run_timed: scan_events is a ctypes array of two hipEvent_t (or None)."""
        o = Outputs()
        for k in INT_FIELDS + ("flags", "reward"):
            setattr(o, k, out[k].data_ptr())
        for k in OPTIONAL_FIELDS:
            setattr(o, k, out[k].data_ptr() if k in out and out[k] is not None else None)
        ev = ctypes.cast(scan_events, ctypes.c_void_p) if scan_events is not None else None
        return lib().parason_run_timed(self._h, tokens_ptr, starts_ptr, lengths_ptr, correct_ptr, int(n_traj),
                                       ctypes.byref(o), ws_ptr, int(ws_bytes), stream, ev)

    def decode_step_raw(self, states_ptr, tokens_ptr, batch, logits_ptr, vocab, row_stride, dtype, eos_id,
                        stream) -> int:
        """Direct parason_decode_step call with raw device pointers; returns the status."""
        return lib().parason_decode_step(self._h, states_ptr, tokens_ptr, int(batch), logits_ptr, int(vocab),
                                         int(row_stride), int(dtype), int(eos_id), stream)

    def decode_step(self, states, logits, tokens=None, eos_id: int = -1):
        """Advance the decode states by `tokens` (int32[batch] or None) and mask
        `logits` ([batch, vocab] rows, float32/bfloat16/float16, unit stride
        along the vocabulary) in place, on the current stream."""
        import torch

        dtypes = {torch.float32: DTYPE_F32, torch.bfloat16: DTYPE_BF16, torch.float16: DTYPE_F16}
        if logits.dtype not in dtypes or logits.dim() != 2 or logits.stride(1) != 1 or not logits.is_cuda:
            raise TypeError("logits must be a [batch, vocab] float32/bfloat16/float16 device tensor, unit stride")
        batch, vocab = logits.shape
        if states.dtype != torch.uint8 or states.numel() != batch * DECODE_STATE_BYTES or not states.is_contiguous():
            raise TypeError("states must be a contiguous uint8 device tensor of batch * 16 bytes")
        if tokens is not None and (tokens.dtype != torch.int32 or tokens.numel() != batch
                                   or not tokens.is_contiguous()):
            raise TypeError("tokens must be a contiguous int32 device tensor of batch entries")
        stream = torch.cuda.current_stream(logits.device).cuda_stream
        rc = self.decode_step_raw(states.data_ptr(), tokens.data_ptr() if tokens is not None else None, batch,
                                  logits.data_ptr(), vocab, logits.stride(0) if batch > 1 else vocab,
                                  dtypes[logits.dtype], eos_id, stream)
        if rc != OK:
            raise ParasonError(rc, "parason_decode_step")
        return logits

    def fork_raw(self, tokens_ptr, starts_ptr, lengths_ptr, n_rows, flags, out: ForkOutputs, ws_ptr, ws_bytes,
                 stream) -> int:
        return lib().parason_fork(self._h, tokens_ptr, starts_ptr, lengths_ptr, int(n_rows), int(flags),
                                  ctypes.byref(out), ws_ptr, int(ws_bytes), stream)

    def join_raw(self, tokens_ptr, starts_ptr, lengths_ptr, n_rows, worker_off_ptr, wtokens_ptr, wstarts_ptr,
                 wlengths_ptr, n_workers, flags, out: JoinOutputs, ws_ptr, ws_bytes, stream) -> int:
        return lib().parason_join(self._h, tokens_ptr, starts_ptr, lengths_ptr, int(n_rows), worker_off_ptr,
                                  wtokens_ptr, wstarts_ptr, wlengths_ptr, int(n_workers), int(flags),
                                  ctypes.byref(out), ws_ptr, int(ws_bytes), stream)

    def fork(self, tokens, starts, lengths, seed: bool = True, max_workers=None, ctx_capacity=None) -> dict:
        """Worker contexts of a batch of rows (device tensors).  Without
        capacities, a first call sizes the outputs (one synchronisation)."""
        import torch

        _check_rows(tokens, starts, lengths)
        dev, n = starts.device, int(starts.numel())
        flags = FORK_SEED_ENTRY if seed else 0
        ws = torch.empty(_ws_size("parason_fork_workspace_size", n), dtype=torch.uint8, device=dev)
        stream = torch.cuda.current_stream(dev).cuda_stream
        i64 = dict(dtype=torch.int64, device=dev)
        i32 = dict(dtype=torch.int32, device=dev)
        res = dict(worker_off=torch.empty(n + 1, **i64), row_status=torch.empty(max(n, 1), **i32)[:n],
                   totals=torch.empty(3, **i64))

        def call(W, T):
            res.update(ctx_tokens=torch.empty(max(T, 1), **i32)[:T], ctx_starts=torch.empty(max(W, 1), **i64)[:W],
                       ctx_lengths=torch.empty(max(W, 1), **i32)[:W], ctx_row=torch.empty(max(W, 1), **i32)[:W],
                       ctx_entry=torch.empty(max(W, 1), **i32)[:W], ctx_kind=torch.empty(max(W, 1), **i32)[:W])
            o = ForkOutputs(int(W), int(T), *[res[k].data_ptr() for k in (
                "ctx_tokens", "ctx_starts", "ctx_lengths", "ctx_row", "ctx_entry", "ctx_kind", "worker_off",
                "row_status", "totals")])
            rc = self.fork_raw(_ptr(tokens, starts), starts.data_ptr(), lengths.data_ptr(), n, flags, o,
                               ws.data_ptr(), ws.numel(), stream)
            if rc != OK:
                raise ParasonError(rc, "parason_fork")

        if max_workers is None or ctx_capacity is None:
            call(0, 0)
            W, T, _ = (int(x) for x in res["totals"].cpu())
            max_workers = W if max_workers is None else max_workers
            ctx_capacity = T if ctx_capacity is None else ctx_capacity
        call(max_workers, ctx_capacity)
        return res

    def join(self, tokens, starts, lengths, worker_off, wtokens, wstarts, wlengths, close: bool = True,
             append_only: bool = False, capacity=None) -> dict:
        """Joined rows (device tensors); sizing as for fork."""
        import torch

        _check_rows(tokens, starts, lengths)
        _check_rows(wtokens, wstarts, wlengths)
        dev, n, nw = starts.device, int(starts.numel()), int(wstarts.numel())
        flags = (JOIN_CLOSE_PARALLEL if close else 0) | (JOIN_APPEND_ONLY if append_only else 0)
        ws = torch.empty(_ws_size("parason_join_workspace_size", n), dtype=torch.uint8, device=dev)
        stream = torch.cuda.current_stream(dev).cuda_stream
        res = dict(starts=torch.empty(n + 1, dtype=torch.int64, device=dev),
                   lengths=torch.empty(max(n, 1), dtype=torch.int32, device=dev)[:n],
                   row_status=torch.empty(max(n, 1), dtype=torch.int32, device=dev)[:n],
                   totals=torch.empty(2, dtype=torch.int64, device=dev))

        def call(T):
            res["tokens"] = torch.empty(max(T, 1), dtype=torch.int32, device=dev)[:T]
            o = JoinOutputs(int(T), *[res[k].data_ptr() for k in ("tokens", "starts", "lengths", "row_status",
                                                                   "totals")])
            rc = self.join_raw(_ptr(tokens, starts), starts.data_ptr(), lengths.data_ptr(), n,
                               worker_off.data_ptr(), _ptr(wtokens, wstarts), wstarts.data_ptr(),
                               wlengths.data_ptr(), nw, flags, o, ws.data_ptr(), ws.numel(), stream)
            if rc != OK:
                raise ParasonError(rc, "parason_join")

        if capacity is None:
            call(0)
            capacity = int(res["totals"][0].item())
        call(capacity)
        return res

    def run(self, tokens, starts, lengths, correct, out: dict | None = None, workspace=None, total_tokens=None,
            derived: bool = True, metrics: bool = False) -> dict:
        """Evaluate a batch of rows held in device tensors (asynchronous on the
        current stream).  tokens int32, starts int64, lengths int32, correct uint8."""
        import torch

        n = int(starts.numel())
        for t, dt in ((tokens, torch.int32), (starts, torch.int64), (lengths, torch.int32), (correct, torch.uint8)):
            if t.dtype != dt or not t.is_cuda or not t.is_contiguous():
                raise TypeError("expected contiguous %s device tensors" % dt)
        if lengths.numel() != n or correct.numel() != n:
            raise ValueError("starts, lengths and correct must have the same length")
        if out is None:
            out = self.alloc_outputs(n, tokens.device, derived, metrics)
        if workspace is None:
            if total_tokens is None:
                total_tokens = int(lengths.to(torch.int64).clamp_min(0).sum().item()) if n else 0
            workspace = self.alloc_workspace(n, total_tokens, tokens.device)
        stream = torch.cuda.current_stream(tokens.device).cuda_stream
        tok_ptr = tokens.data_ptr() if tokens.numel() else starts.data_ptr()
        rc = self.run_raw(tok_ptr, starts.data_ptr(), lengths.data_ptr(), correct.data_ptr(), n, out,
                          workspace.data_ptr(), workspace.numel(), stream)
        if rc != OK:
            raise ParasonError(rc, "parason_run")
        return out


def read_probe_raw(data_ptr, nbytes, sink_ptr, sink_len, stream) -> int:
    """parason_read_probe: streaming read of nbytes at data_ptr (measurement)."""
    return lib().parason_read_probe(data_ptr, int(nbytes), sink_ptr, int(sink_len), stream)


def _check_rows(tokens, starts, lengths):
    import torch

    for t, dt in ((tokens, torch.int32), (starts, torch.int64), (lengths, torch.int32)):
        if t.dtype != dt or not t.is_cuda or not t.is_contiguous():
            raise TypeError("expected contiguous %s device tensors" % dt)
    if starts.numel() != lengths.numel():
        raise ValueError("starts and lengths must have the same length")


def _ptr(tokens, fallback):
    return tokens.data_ptr() if tokens.numel() else fallback.data_ptr()


def _ws_size(name: str, n: int) -> int:
    b = ctypes.c_size_t()
    rc = getattr(lib(), name)(int(n), ctypes.byref(b))
    if rc != OK:
        raise ParasonError(rc, name)
    return b.value


def decode_init(batch: int, device, states=None):
    """Decode states (uint8[batch * 16] device tensor) set to the start of a stream."""
    import torch

    if states is None:
        states = torch.empty(int(batch) * DECODE_STATE_BYTES, dtype=torch.uint8, device=device)
    stream = torch.cuda.current_stream(states.device).cuda_stream
    rc = lib().parason_decode_init(states.data_ptr(), int(batch), stream)
    if rc != OK:
        raise ParasonError(rc, "parason_decode_init")
    return states


def decode_fields(states):
    """[batch, 4] int32 view of a states tensor: state, depth, entry, flags."""
    import torch

    return states.view(torch.int32).view(-1, 4)


def pg_workspace_size(n_traj: int) -> int:
    b = ctypes.c_size_t()
    rc = lib().parason_pg_workspace_size(int(n_traj), ctypes.byref(b))
    if rc != OK:
        raise ParasonError(rc, "parason_pg_workspace_size")
    return b.value


def pg_run_raw(cfg: PgConfig, reward_ptr, logp_ptr, old_ptr, starts_ptr, lengths_ptr, n_traj, adv_ptr, grad_ptr,
               stats_ptr, ws_ptr, ws_bytes, stream) -> int:
    return lib().parason_pg_run(ctypes.byref(cfg), reward_ptr, logp_ptr, old_ptr, starts_ptr, lengths_ptr,
                                int(n_traj), adv_ptr, grad_ptr, stats_ptr, ws_ptr, int(ws_bytes), stream)


def pg_run(reward, logp, logp_old, starts, lengths, group_size=8, clip_low=0.2, clip_high=0.28, grad=None,
           workspace=None) -> dict:
    """Advantages, gradient d loss / d logp and the step statistics (device
    tensors; asynchronous on the current stream).  reward float32[n], logp and
    logp_old float32 in the row layout of starts/lengths."""
    import torch

    n = int(starts.numel())
    for t, dt in ((reward, torch.float32), (logp, torch.float32), (logp_old, torch.float32),
                  (starts, torch.int64), (lengths, torch.int32)):
        if t.dtype != dt or not t.is_cuda or not t.is_contiguous():
            raise TypeError("expected contiguous %s device tensors" % dt)
    dev = logp.device
    cfg = PgConfig(int(group_size), float(clip_low), float(clip_high))
    adv = torch.empty(n, dtype=torch.float32, device=dev)
    if grad is None:
        grad = torch.empty_like(logp)
    stats = torch.empty(len(PG_STATS), dtype=torch.float64, device=dev)
    if workspace is None:
        workspace = torch.empty(pg_workspace_size(n), dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream(dev).cuda_stream
    rc = pg_run_raw(cfg, reward.data_ptr(), logp.data_ptr(), logp_old.data_ptr(), starts.data_ptr(),
                    lengths.data_ptr(), n, adv.data_ptr(), grad.data_ptr(), stats.data_ptr(), workspace.data_ptr(),
                    workspace.numel(), stream)
    if rc != OK:
        raise ParasonError(rc, "parason_pg_run")
    return dict(advantage=adv, grad=grad, stats=stats)
