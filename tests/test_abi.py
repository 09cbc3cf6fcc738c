"""C-ABI checks that need no GPU: the library loads, exports every function the
header declares, and rejects bad arguments on the host before any launch.

Every parason_run call here fails a host-side check before the first HIP call,
so these tests are safe on a GPU machine too (no kernel ever sees the fake
pointers)."""
import ctypes
import os
import re

import pytest

from paper_2608_24658_amd import parason as P

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "parason.h")
TAGS = list(range(151924, 151936))
FAKE = 0x100000  # never dereferenced: each call below fails a host check first


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(parason_[a-z_]+)\s*\(", src)))


def test_exports_every_declared_function():
    names = declared_functions()
    assert set(names) == set(P.EXPORTED)
    L = P.lib()
    for n in names:
        assert hasattr(L, n), n


def test_strerror_covers_codes():
    for rc in range(0, -11, -1):
        assert P.strerror(rc) != "unknown status"
    assert P.strerror(-99) == "unknown status"


def _create(cfg):
    h = ctypes.c_void_p()
    rc = P.lib().parason_create(ctypes.byref(cfg), ctypes.byref(h))
    if rc == P.OK:
        P.lib().parason_destroy(h)
    return rc


def test_create_validates_config():
    assert _create(P.make_config(TAGS)) == P.OK
    assert _create(P.make_config(TAGS[:11] + [TAGS[0]])) == P.ERR_TAGS
    assert _create(P.make_config([-1] + TAGS[1:])) == P.ERR_TAGS
    assert _create(P.make_config(TAGS, group_size=0)) == P.ERR_GROUP
    assert _create(P.make_config(TAGS, alpha=float("nan"))) == P.ERR_PARAM
    assert _create(P.make_config(TAGS, rho_clip=float("inf"))) == P.ERR_PARAM
    h = ctypes.c_void_p()
    assert P.lib().parason_create(None, ctypes.byref(h)) == P.ERR_NULL
    with pytest.raises(P.ParasonError):
        P.Parason(TAGS, group_size=-3)


def test_workspace_size_validates_and_grows():
    px = P.Parason(TAGS)
    a = px.workspace_size(8, 1000)
    b = px.workspace_size(8, 10 ** 6)
    c = px.workspace_size(800, 10 ** 6)
    assert 0 < a < b < c
    # about 56 bytes per 1024-token segment for a large batch (1.4 % of the token bytes)
    big = px.workspace_size(712000, 35825658097)
    assert big < 0.015 * 4 * 35825658097
    # slot indices are 32-bit: beyond about 3.6e11 tokens the size is refused
    assert px.workspace_size(8, 3 * 10 ** 11) > 0
    with pytest.raises(P.ParasonError):
        px.workspace_size(8, 4 * 10 ** 11)
    with pytest.raises(P.ParasonError):
        px.workspace_size(-1, 10)
    with pytest.raises(P.ParasonError):
        px.workspace_size(8, -10)
    sz = ctypes.c_size_t()
    assert P.lib().parason_workspace_size(None, 8, 10, ctypes.byref(sz)) == P.ERR_NULL


class _FakeOut(dict):
    def __init__(self):
        class T:
            def __init__(self, p):
                self.p = p

            def data_ptr(self):
                return self.p

        super().__init__({k: T(FAKE) for k in P.INT_FIELDS + ("flags", "reward")})


def test_run_rejects_bad_arguments_before_launch():
    px = P.Parason(TAGS, group_size=8)
    out = _FakeOut()
    ws = px.workspace_size(16, 1000)
    run = px.run_raw
    # n_traj not a multiple of G
    assert run(FAKE, FAKE, FAKE, FAKE, 12, out, FAKE, ws, None) == P.ERR_GROUP
    assert run(FAKE, FAKE, FAKE, FAKE, -8, out, FAKE, ws, None) == P.ERR_SIZE
    # n_traj == 0 is a no-op
    assert run(0, 0, 0, 0, 0, out, 0, 0, None) == P.OK
    # NULL inputs
    assert run(0, FAKE, FAKE, FAKE, 16, out, FAKE, ws, None) == P.ERR_NULL
    assert run(FAKE, FAKE, FAKE, 0, 16, out, FAKE, ws, None) == P.ERR_NULL
    assert run(FAKE, FAKE, FAKE, FAKE, 16, out, 0, ws, None) == P.ERR_NULL
    bad = dict(out)
    bad["reward"] = type(out["reward"])(0)
    assert run(FAKE, FAKE, FAKE, FAKE, 16, bad, FAKE, ws, None) == P.ERR_NULL
    # alignment: tokens must be 4-byte aligned, the workspace 256-byte aligned
    assert run(FAKE + 2, FAKE, FAKE, FAKE, 16, out, FAKE, ws, None) == P.ERR_ALIGN
    assert run(FAKE, FAKE, FAKE, FAKE, 16, out, FAKE + 64, ws, None) == P.ERR_ALIGN
    # workspace too small
    assert run(FAKE, FAKE, FAKE, FAKE, 16, out, FAKE, 1024, None) == P.ERR_WORKSPACE
    assert P.lib().parason_run(None, FAKE, FAKE, FAKE, FAKE, 16, None, FAKE, ws, None) == P.ERR_NULL


def test_decode_rejects_bad_arguments_before_launch():
    px = P.Parason(TAGS)
    V = 151936
    step = px.decode_step_raw
    bf = P.DTYPE_BF16
    assert P.lib().parason_decode_step(None, FAKE, FAKE, 4, FAKE, V, V, bf, 0, None) == P.ERR_NULL
    assert step(FAKE, FAKE, -1, FAKE, V, V, bf, 0, None) == P.ERR_SIZE
    assert step(FAKE, FAKE, 4, FAKE, 0, 0, bf, 0, None) == P.ERR_SIZE
    assert step(FAKE, FAKE, 4, FAKE, V, V - 1, bf, 0, None) == P.ERR_SIZE
    assert step(FAKE, FAKE, 4, FAKE, V, V, 7, 0, None) == P.ERR_PARAM
    # every tag id and the eos id must be inside the vocabulary; eos is no tag
    assert step(FAKE, FAKE, 4, FAKE, TAGS[-1], TAGS[-1], bf, 0, None) == P.ERR_TAGS
    assert step(FAKE, FAKE, 4, FAKE, V, V, bf, TAGS[3], None) == P.ERR_TAGS
    assert step(FAKE, FAKE, 4, FAKE, V, V, bf, V, None) == P.ERR_TAGS
    assert step(FAKE, FAKE, 4, FAKE, V, V, bf, -2, None) == P.ERR_TAGS
    # batch 0 is a no-op; NULL and misaligned pointers
    assert step(0, 0, 0, 0, V, V, bf, 0, None) == P.OK
    assert step(0, FAKE, 4, FAKE, V, V, bf, 0, None) == P.ERR_NULL
    assert step(FAKE, FAKE, 4, 0, V, V, bf, 0, None) == P.ERR_NULL
    assert step(FAKE + 4, FAKE, 4, FAKE, V, V, bf, 0, None) == P.ERR_ALIGN
    assert step(FAKE, FAKE, 4, FAKE + 1, V, V, bf, 0, None) == P.ERR_ALIGN
    assert step(FAKE, FAKE, 4, FAKE + 2, V, V, P.DTYPE_F32, 0, None) == P.ERR_ALIGN
    assert step(FAKE, FAKE + 2, 4, FAKE, V, V, bf, 0, None) == P.ERR_ALIGN
    init = P.lib().parason_decode_init
    assert init(None, 4, None) == P.ERR_NULL
    assert init(FAKE, -1, None) == P.ERR_SIZE
    assert init(FAKE + 8, 4, None) == P.ERR_ALIGN
    assert init(None, 0, None) == P.OK


def test_fork_join_reject_bad_arguments_before_launch():
    px = P.Parason(TAGS)
    ws = ctypes.c_size_t()
    assert P.lib().parason_fork_workspace_size(16, ctypes.byref(ws)) == P.OK and ws.value > 0
    assert P.lib().parason_fork_workspace_size(-1, ctypes.byref(ws)) == P.ERR_SIZE
    assert P.lib().parason_join_workspace_size(16, None) == P.ERR_NULL
    P.lib().parason_fork_workspace_size(16, ctypes.byref(ws))
    W = ws.value
    fo = P.ForkOutputs(4, 100, *([FAKE] * 9))
    fork = px.fork_raw
    assert P.lib().parason_fork(None, FAKE, FAKE, FAKE, 16, 0, ctypes.byref(fo), FAKE, W, None) == P.ERR_NULL
    assert fork(FAKE, FAKE, FAKE, -1, 0, fo, FAKE, W, None) == P.ERR_SIZE
    assert fork(FAKE, FAKE, FAKE, 16, 4, fo, FAKE, W, None) == P.ERR_PARAM
    assert fork(0, FAKE, FAKE, 16, 0, fo, FAKE, W, None) == P.ERR_NULL
    assert fork(FAKE, FAKE, FAKE, 16, 0, fo, 0, W, None) == P.ERR_NULL
    assert fork(FAKE + 2, FAKE, FAKE, 16, 0, fo, FAKE, W, None) == P.ERR_ALIGN
    assert fork(FAKE, FAKE, FAKE, 16, 0, fo, FAKE + 8, W, None) == P.ERR_ALIGN
    assert fork(FAKE, FAKE, FAKE, 16, 0, fo, FAKE, W - 1, None) == P.ERR_WORKSPACE
    for k in ("ctx_tokens", "ctx_starts", "ctx_kind", "worker_off", "row_status", "totals"):
        bad = P.ForkOutputs(4, 100, *([FAKE] * 9))
        setattr(bad, k, None)
        assert fork(FAKE, FAKE, FAKE, 16, 0, bad, FAKE, W, None) == P.ERR_NULL, k
    neg = P.ForkOutputs(-1, 100, *([FAKE] * 9))
    assert fork(FAKE, FAKE, FAKE, 16, 0, neg, FAKE, W, None) == P.ERR_SIZE
    P.lib().parason_join_workspace_size(16, ctypes.byref(ws))
    W = ws.value
    jo = P.JoinOutputs(100, *([FAKE] * 5))
    join = px.join_raw
    assert join(FAKE, FAKE, FAKE, 16, FAKE, FAKE, FAKE, FAKE, 32, 4, jo, FAKE, W, None) == P.ERR_PARAM
    assert join(FAKE, FAKE, FAKE, 16, FAKE, FAKE, FAKE, FAKE, -1, 0, jo, FAKE, W, None) == P.ERR_SIZE
    assert join(FAKE, FAKE, FAKE, 16, 0, FAKE, FAKE, FAKE, 32, 0, jo, FAKE, W, None) == P.ERR_NULL
    assert join(FAKE, FAKE, FAKE, 16, FAKE, 0, FAKE, FAKE, 32, 0, jo, FAKE, W, None) == P.ERR_NULL
    assert join(FAKE, FAKE, FAKE, 16, FAKE, FAKE + 1, FAKE, FAKE, 32, 0, jo, FAKE, W, None) == P.ERR_ALIGN
    assert join(FAKE, FAKE, FAKE, 16, FAKE, FAKE, FAKE, FAKE, 32, 0, jo, FAKE, 64, None) == P.ERR_WORKSPACE
    bad = P.JoinOutputs(100, None, FAKE, FAKE, FAKE, FAKE)
    assert join(FAKE, FAKE, FAKE, 16, FAKE, FAKE, FAKE, FAKE, 32, 0, bad, FAKE, W, None) == P.ERR_NULL


def _gpu_visible():
    """True when a HIP device is visible (counting devices does not initialise one)."""
    try:
        import torch

        return torch.cuda.device_count() > 0
    except Exception:
        return False


@pytest.mark.skipif(_gpu_visible(), reason="with a GPU these calls would pass the device check and launch")
def test_launching_calls_check_the_device_first():
    """With no gfx950 device current, every call that launches returns
    PARASON_ERR_DEVICE after its argument checks and before any launch (the
    fake pointers are never dereferenced)."""
    px = P.Parason(TAGS, group_size=8)
    out = _FakeOut()
    ws = px.workspace_size(16, 1000)
    assert px.run_raw(FAKE, FAKE, FAKE, FAKE, 16, out, FAKE, ws, None) == P.ERR_DEVICE
    assert P.lib().parason_decode_init(FAKE, 4, None) == P.ERR_DEVICE
    V = 151936
    assert px.decode_step_raw(FAKE, FAKE, 4, FAKE, V, V, P.DTYPE_BF16, 0, None) == P.ERR_DEVICE
    pw = ctypes.c_size_t()
    assert P.lib().parason_pg_workspace_size(16, ctypes.byref(pw)) == P.OK
    cfg = P.PgConfig(8, 0.2, 0.28)
    assert P.pg_run_raw(cfg, FAKE, FAKE, FAKE, FAKE, FAKE, 16, FAKE, FAKE, FAKE, FAKE, pw.value, None) == P.ERR_DEVICE
    fw = ctypes.c_size_t()
    P.lib().parason_fork_workspace_size(16, ctypes.byref(fw))
    fo = P.ForkOutputs(4, 100, *([FAKE] * 9))
    assert px.fork_raw(FAKE, FAKE, FAKE, 16, 0, fo, FAKE, fw.value, None) == P.ERR_DEVICE
    jw = ctypes.c_size_t()
    P.lib().parason_join_workspace_size(16, ctypes.byref(jw))
    jo = P.JoinOutputs(100, *([FAKE] * 5))
    assert px.join_raw(FAKE, FAKE, FAKE, 16, FAKE, FAKE, FAKE, FAKE, 32, 0, jo, FAKE, jw.value, None) == P.ERR_DEVICE
    assert P.read_probe_raw(FAKE, 4096, FAKE, 1, None) == P.ERR_DEVICE
    assert px.run_noalloc_raw(FAKE, FAKE, FAKE, FAKE, 16, 1000, out, None) == P.ERR_DEVICE


def test_read_probe_rejects_bad_arguments_before_launch():
    rp = P.read_probe_raw
    assert rp(0, 0, 0, 0, None) == P.OK  # nothing to read
    assert rp(0, 4096, FAKE, 1, None) == P.ERR_NULL
    assert rp(FAKE, 4096, 0, 1, None) == P.ERR_NULL
    assert rp(FAKE, 4096, FAKE, 0, None) == P.ERR_SIZE
    assert rp(FAKE, 4095, FAKE, 1, None) == P.ERR_SIZE
    assert rp(FAKE + 4, 4096, FAKE, 1, None) == P.ERR_ALIGN
    assert rp(FAKE, 4096, FAKE + 2, 1, None) == P.ERR_ALIGN


def test_run_noalloc_rejects_bad_arguments_before_launch():
    """parason_run_noalloc: argument errors, and a batch whose workspace would
    exceed the static scratch, are refused on the host."""
    px = P.Parason(TAGS, group_size=8)
    out = _FakeOut()
    run = px.run_noalloc_raw
    assert run(0, 0, 0, 0, 0, 0, out, None) == P.OK  # nothing to do
    assert run(FAKE, FAKE, FAKE, FAKE, 12, 1000, out, None) == P.ERR_GROUP
    assert run(FAKE, FAKE, FAKE, FAKE, -8, 1000, out, None) == P.ERR_SIZE
    assert run(FAKE, FAKE, FAKE, FAKE, 16, -1, out, None) == P.ERR_SIZE
    assert P.lib().parason_run_noalloc(None, FAKE, FAKE, FAKE, FAKE, 16, 1000, None, None) == P.ERR_NULL
    # the largest token count whose workspace fits, and one segment's worth more
    lo, hi = 0, 1 << 36
    while hi - lo > 1:
        mid = (lo + hi) // 2
        lo, hi = (mid, hi) if px.workspace_size(16, mid) <= P.NOALLOC_SCRATCH_BYTES else (lo, mid)
    assert px.workspace_size(16, lo) <= P.NOALLOC_SCRATCH_BYTES < px.workspace_size(16, lo + 4096)
    assert run(FAKE, FAKE, FAKE, FAKE, 16, lo + 4096, out, None) == P.ERR_SCRATCH
    assert run(FAKE, FAKE, FAKE, FAKE, 16, 10 ** 11, out, None) == P.ERR_SCRATCH
    # beyond what any workspace can index (3.6e11 tokens): a size error
    assert run(FAKE, FAKE, FAKE, FAKE, 16, 10 ** 12, out, None) == P.ERR_SIZE
    assert "scratch" in P.strerror(P.ERR_SCRATCH)
