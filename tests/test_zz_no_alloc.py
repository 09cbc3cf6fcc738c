"""parason_run_noalloc (the entry point for callers that cannot allocate:
its scratch is the library's static device array) against parason_run on
the same inputs, through the C-ABI: two calls in a row, the second with a
smaller batch, every output bit for bit; then a batch beyond the scratch is
refused before any launch.  Runs on its own in a fresh process and after the
other tests (the scratch keeps the previous call's contents; no call relies
on them)."""
import numpy as np
import pytest

from gpu_util import DEFAULT_COEF, fetch, log
from paper_2608_24658_amd import parason as PX
from paper_2608_24658_amd.synth import synth as S

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

G = S.GROUP_SIZE


def run_both(px, dev, workload, flags_note):
    P = S.make_params(workload)
    n = S.n_rows_of(workload)
    tok, st, ln, co = S.device_batch(P, n, device=dev)
    total = int(tok.numel())
    stream = torch.cuda.current_stream(dev).cuda_stream
    ref = px.run(tok, st, ln, co, total_tokens=total)  # parason_run with a workspace
    out = px.alloc_outputs(n, dev)
    for v in out.values():
        v.fill_(-7)  # any value the call must overwrite
    log("case no-alloc %s: %d rows, %d tokens (%s)" % (workload, n, total, flags_note))
    rc = px.run_noalloc_raw(tok.data_ptr(), st.data_ptr(), ln.data_ptr(), co.data_ptr(), n, total, out, stream)
    assert rc == PX.OK, PX.strerror(rc)
    torch.cuda.synchronize()
    a, b = fetch(ref), fetch(out)
    for k in a:
        assert np.array_equal(a[k].view(np.uint32) if a[k].dtype == np.float32 else a[k],
                              b[k].view(np.uint32) if b[k].dtype == np.float32 else b[k]), (workload, k)
    assert np.all(a["flags"] & PX.FLAG_VALID) or workload == "ragged"
    return n


@pytest.mark.parametrize("lenient", [False, True])
def test_noalloc_matches_run(lenient):
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    dev = torch.device("cuda:0")
    px = PX.Parason(S.CONTIGUOUS_TAGS, group_size=G, flags=PX.CFG_LENIENT_GAPS if lenient else 0, **DEFAULT_COEF)
    # the typical batch (2,048 rows, 9.3e7 tokens) fills most of the scratch;
    # the smaller batches after it run on what it left there
    for wl in ("typical", "small", "ragged", "tiny"):
        run_both(px, dev, wl, "lenient" if lenient else "strict")
    # beyond the scratch: refused on the host
    out = px.alloc_outputs(G, dev)
    t = torch.zeros(16, dtype=torch.int32, device=dev)
    rc = px.run_noalloc_raw(t.data_ptr(), t.data_ptr(), t.data_ptr(), t.data_ptr(), G, 10 ** 11, out,
                            torch.cuda.current_stream(dev).cuda_stream)
    assert rc == PX.ERR_SCRATCH
