"""GPU parity: the HIP path (through the C-ABI) against the CPU oracle.

Inputs are the seeded synthetic workloads (generated on the device and
regenerated bit-identically by the host mirror) and hand-built adversarial
batches.  Integer outputs must be bit-exact; float outputs the float rounding
of the oracle's double values (see gpu_util).
"""
import numpy as np
import pytest

import grammar_pins as GP
from adversarial import adversarial_streams, deep_stream, pack
from gpu_util import DEFAULT_COEF, compare, fetch, log, oracle_expect, run_gpu, to_dev
from oracle import oracle as O
from paper_2608_24658_amd import parason as PX
from paper_2608_24658_amd.synth import synth as S

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

G = S.GROUP_SIZE
TAGS = S.CONTIGUOUS_TAGS


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch.device("cuda:0")


# twelve of the ids 0..15, not consecutive: the scan's hash separates them while
# the text ids next to them (5, 7, 12, 14) land in slots of their own
LOW_IDS = np.array([3, 9, 4, 11, 0, 13, 1, 6, 15, 2, 10, 8], dtype=np.int32)


def px_for(tags=TAGS, flags=0, **kw):
    coef = dict(DEFAULT_COEF)
    coef.update(kw)
    return PX.Parason(tags, group_size=G, flags=flags, **coef), coef


@pytest.mark.parametrize("workload", ["tiny", "small", "ragged", "typical"])
def test_workload_parity(dev, workload):
    log("case workload=%s" % workload)
    P = S.make_params(workload)
    n = S.n_rows_of(workload)
    tok_d, st_d, ln_d, co_d = S.device_batch(P, n, device=dev)
    tok_h, st_h, ln_h, co_h = S.host_batch(P, n)
    assert np.array_equal(st_d.cpu().numpy(), st_h) and np.array_equal(ln_d.cpu().numpy(), ln_h)
    assert np.array_equal(co_d.cpu().numpy(), co_h)
    assert np.array_equal(tok_d.cpu().numpy(), tok_h), "device generator differs from the host mirror"
    px, coef = px_for()
    got = run_gpu(px, tok_d, st_d, ln_d, co_d)
    rows, R, rs, rt, eta = oracle_expect(tok_h, st_h, ln_h, co_h, TAGS, G, coef)
    n_exact = compare(got, rows, R, rs, rt, eta, what=workload)
    log("%s: %d rows, %d tokens, %d/%d rewards bit-exact" % (workload, n, tok_h.size, n_exact, n))


@pytest.mark.parametrize("tag_test", ["hash", "compare"])
def test_scattered_tag_ids(dev, tag_test):
    """Tag ids that are not twelve consecutive values: the scan's hashed lookup
    and, with PARASON_CFG_TAG_COMPARE, its twelve-compare test."""
    log("case scattered tags %s" % tag_test)
    P = S.make_params("small", tag_ids=S.SCATTERED_TAGS)
    n = S.n_rows_of("small")
    tok_d, st_d, ln_d, co_d = S.device_batch(P, n, device=dev)
    tok_h, st_h, ln_h, co_h = S.host_batch(P, n)
    assert np.array_equal(tok_d.cpu().numpy(), tok_h)
    flags = PX.CFG_TAG_COMPARE if tag_test == "compare" else 0
    px, coef = px_for(S.SCATTERED_TAGS, flags=flags, alpha=0.0, beta_subtask=0.05, beta_trial=0.0)
    got = run_gpu(px, tok_d, st_d, ln_d, co_d)
    compare(got, *oracle_expect(tok_h, st_h, ln_h, co_h, S.SCATTERED_TAGS, G, coef), what="scattered")


@pytest.mark.parametrize("tags", ["contiguous", "scattered", "scattered-compare", "low-ids"])
def test_adversarial_streams(dev, tags):
    log("case adversarial tags=%s" % tags)
    tag_ids = {"contiguous": TAGS, "low-ids": LOW_IDS}.get(tags, S.SCATTERED_TAGS)
    tokens, starts, lengths = pack(adversarial_streams(), tag_ids)
    n = lengths.size
    correct = (np.arange(n) % 3 != 0).astype(np.uint8)
    px, coef = px_for(tag_ids, flags=PX.CFG_TAG_COMPARE if tags == "scattered-compare" else 0)
    got = run_gpu(px, to_dev(tokens, torch.int32, dev), to_dev(starts, torch.int64, dev),
                  to_dev(lengths, torch.int32, dev), to_dev(correct, torch.uint8, dev))
    compare(got, *oracle_expect(tokens, starts, lengths, correct, tag_ids, G, coef), what="adversarial")
    assert int(np.sum(got["max_depth"] == 1000)) == 1
    log("adversarial: %d rows ok" % n)


@pytest.mark.parametrize("reps", [4, 18])
@pytest.mark.parametrize("tags", ["scattered", "scattered-compare", "low-ids"])
def test_tag_lookups_on_the_larger_batch_paths(dev, tags, reps):
    """The hashed and the twelve-compare tag tests in the scan instances and row
    kernels of batches the scan does not plan itself: the adversarial rows
    repeated 4 times (2,392 rows: the plan launch, then rows_par) and 18 times
    (10,768 rows with the padding to whole groups: the per-lane row tiers,
    their gather and the deep tier)."""
    log("case tag lookups tags=%s reps=%d" % (tags, reps))
    tag_ids = {"low-ids": LOW_IDS}.get(tags, S.SCATTERED_TAGS)
    tokens, starts, lengths = pack(adversarial_streams() * reps, tag_ids)
    n = lengths.size
    assert (n > 2048) and ((n >= 10240) == (reps == 18))
    correct = (np.arange(n) % 3 != 2).astype(np.uint8)
    px, coef = px_for(tag_ids, flags=PX.CFG_TAG_COMPARE if tags == "scattered-compare" else 0)
    got = run_gpu(px, to_dev(tokens, torch.int32, dev), to_dev(starts, torch.int64, dev),
                  to_dev(lengths, torch.int32, dev), to_dev(correct, torch.uint8, dev))
    compare(got, *oracle_expect(tokens, starts, lengths, correct, tag_ids, G, coef), what="tag lookups")
    assert int(np.sum(got["max_depth"] == 1000)) == reps
    log("tag lookups: %d rows ok" % n)


@pytest.mark.parametrize("n", [0, 8, 2056, 10240])
def test_batches_without_tokens(dev, n):
    """Degenerate batches: no rows, and rows that are all empty (not one token
    in the batch) on each batch path: the scan's own plan (8 rows), the plan
    launch with rows_par (2,056), the per-lane row tiers (10,240)."""
    log("case batch without tokens n=%d" % n)
    tokens = np.zeros(0, np.int32)
    starts = np.zeros(n, np.int64)
    lengths = np.zeros(n, np.int32)
    correct = (np.arange(n) % 2).astype(np.uint8)
    px, coef = px_for()
    got = run_gpu(px, to_dev(tokens, torch.int32, dev), to_dev(starts, torch.int64, dev),
                  to_dev(lengths, torch.int32, dev), to_dev(correct, torch.uint8, dev))
    assert all(v.size == n for v in got.values())
    if n:
        compare(got, *oracle_expect(tokens, starts, lengths, correct, TAGS, G, coef), what="no tokens")
        assert np.all(got["total"] == 0)


@pytest.mark.parametrize("tags", ["contiguous", "scattered", "scattered-compare", "low-ids"])
def test_text_ids_over_the_whole_int32_range(dev, tags):
    """Every id that is not one of the twelve tags is Text: negative ids, ids
    just outside a contiguous tag range and the int32 extremes, mixed with
    ids drawn from the whole int32 range (the contiguous scan first compares
    each vector's largest signed token with the first tag id)."""
    log("case text ids over int32 tags=%s" % tags)
    tag_ids = {"contiguous": TAGS, "low-ids": LOW_IDS}.get(tags, S.SCATTERED_TAGS)
    lo, hi = min(tag_ids), max(tag_ids)
    i32 = np.iinfo(np.int32)
    edges = [i32.min, i32.min + 1, -(1 << 24), -2, -1, 0, 1, lo - 1, hi + 1, hi + 2, i32.max - 1, i32.max]
    wide = np.random.default_rng(5).integers(i32.min, i32.max, size=4096, endpoint=True)
    text_ids = np.array([e for e in edges if i32.min <= e <= i32.max] * 64 + list(wide), dtype=np.int64)
    text_ids = text_ids[~np.isin(text_ids, tag_ids)].astype(np.int32)
    tokens, starts, lengths = pack(adversarial_streams(), tag_ids, text_ids=text_ids)
    assert np.any(tokens < 0) and np.any(tokens == i32.max)
    n = lengths.size
    correct = (np.arange(n) % 3 != 1).astype(np.uint8)
    px, coef = px_for(tag_ids, flags=PX.CFG_TAG_COMPARE if tags == "scattered-compare" else 0)
    got = run_gpu(px, to_dev(tokens, torch.int32, dev), to_dev(starts, torch.int64, dev),
                  to_dev(lengths, torch.int32, dev), to_dev(correct, torch.uint8, dev))
    compare(got, *oracle_expect(tokens, starts, lengths, correct, tag_ids, G, coef), what="int32 text ids")
    log("int32 text ids: %d rows ok" % n)


@pytest.mark.parametrize("n", [2040, 2048, 2056, 4104])
def test_plan_boundaries(dev, n):
    """Around the batch sizes where the plan changes: up to 2,048 rows (that
    take rows_par) the scan blocks plan the batch themselves; 2,056 rows take
    the one-block plan launch; 4,104 rows two plan tiles.  Rows of the small
    workload, every output compared with the oracle."""
    log("case plan boundary n=%d" % n)
    P = S.make_params("small")
    tok_h, st_h, ln_h, co_h = S.host_batch(P, n)
    px, coef = px_for()
    got = run_gpu(px, to_dev(tok_h, torch.int32, dev), to_dev(st_h, torch.int64, dev),
                  to_dev(ln_h, torch.int32, dev), to_dev(co_h, torch.uint8, dev))
    compare(got, *oracle_expect(tok_h, st_h, ln_h, co_h, TAGS, G, coef), what="plan boundary %d" % n)


def test_many_rows_beyond_the_first_tier(dev):
    """40,000 rows nested 6-33 deep (more than the second tier has threads, so
    its threads stride over the handed-over list) and 48 rows nested 34-60
    deep (the single-thread tier), mixed with shallow rows."""
    log("case tiers")
    rng = np.random.default_rng(12)
    depths = np.concatenate([rng.integers(6, 34, size=40000), rng.integers(34, 61, size=48),
                             rng.integers(1, 6, size=8000)])
    rng.shuffle(depths)
    streams = [deep_stream(int(d), GP.TRI if d % 2 else GP.SUB) for d in depths]
    tokens, starts, lengths = pack(streams, TAGS)
    n = lengths.size
    correct = (np.arange(n) % 5 != 0).astype(np.uint8)
    px, coef = px_for()
    got = run_gpu(px, to_dev(tokens, torch.int32, dev), to_dev(starts, torch.int64, dev),
                  to_dev(lengths, torch.int32, dev), to_dev(correct, torch.uint8, dev))
    compare(got, *oracle_expect(tokens, starts, lengths, correct, TAGS, G, coef), what="tiers")
    assert np.array_equal(got["max_depth"][: depths.size], depths.astype(np.int32))


def test_layouts_misaligned_padded_overlapping_reversed(dev):
    log("case layouts")
    P = S.make_params("small")
    tok_h, st_h, ln_h, co_h = S.host_batch(P, 64)
    px, coef = px_for()
    expect = oracle_expect(tok_h, st_h, ln_h, co_h, TAGS, G, coef)
    # misaligned base pointer: tokens start 1, 2, 3 elements past a 16-byte boundary
    for shift in (1, 2, 3):
        buf = np.concatenate([np.full(shift, 5, np.int32), tok_h])
        d = to_dev(buf, torch.int32, dev)[shift:]
        got = run_gpu(px, d, to_dev(st_h, torch.int64, dev), to_dev(ln_h, torch.int32, dev),
                      to_dev(co_h, torch.uint8, dev))
        compare(got, *expect, what="shift %d" % shift)
    # padded [B, Lmax] layout with odd Lmax (rows start at every alignment)
    lmax = int(ln_h.max()) + 3
    padded = np.full((64, lmax), 11, np.int32)
    for i in range(64):
        padded[i, : ln_h[i]] = tok_h[st_h[i]: st_h[i] + ln_h[i]]
    starts_p = (np.arange(64) * lmax).astype(np.int64)
    got = run_gpu(px, to_dev(padded.ravel(), torch.int32, dev), to_dev(starts_p, torch.int64, dev),
                  to_dev(ln_h, torch.int32, dev), to_dev(co_h, torch.uint8, dev))
    compare(got, *expect, what="padded")
    # rows in reverse order
    perm = np.arange(64)[::-1].copy()
    got = run_gpu(px, to_dev(tok_h, torch.int32, dev), to_dev(st_h[perm], torch.int64, dev),
                  to_dev(ln_h[perm], torch.int32, dev), to_dev(co_h[perm], torch.uint8, dev))
    rows, R, rs, rt, eta = oracle_expect(tok_h, st_h[perm], ln_h[perm], co_h[perm], TAGS, G, coef)
    compare(got, rows, R, rs, rt, eta, what="reversed")
    # overlapping rows: every row is the same stream, plus prefixes of it
    st_o = np.zeros(64, np.int64)
    ln_o = np.array([ln_h[0] - (i % 5) * 7 for i in range(64)], np.int32)
    got = run_gpu(px, to_dev(tok_h, torch.int32, dev), to_dev(st_o, torch.int64, dev),
                  to_dev(ln_o, torch.int32, dev), to_dev(co_h, torch.uint8, dev))
    compare(got, *oracle_expect(tok_h, st_o, ln_o, co_h, TAGS, G, coef), what="overlapping")


def test_bad_rows_and_workspace_overflow(dev):
    log("case bad rows / overflow")
    P = S.make_params("small")
    tok_h, st_h, ln_h, co_h = S.host_batch(P, 32)
    px, coef = px_for()
    ln_bad = ln_h.copy()
    ln_bad[9] = -5
    got = run_gpu(px, to_dev(tok_h, torch.int32, dev), to_dev(st_h, torch.int64, dev),
                  to_dev(ln_bad, torch.int32, dev), to_dev(co_h, torch.uint8, dev))
    assert got["flags"][9] == PX.FLAG_BAD_ROW
    assert np.all(np.isnan(got["reward"][8:16]))
    keep = np.r_[0:8, 16:32]
    compare({k: v[keep] for k, v in got.items()},
            *oracle_expect(tok_h, st_h[keep], ln_h[keep], co_h[keep], TAGS, G, coef), what="bad-row rest")
    # a workspace sized for no tokens at all, for rows of many segments each
    Pt = S.make_params("typical")
    tok_t, st_t, ln_t, co_t = S.host_batch(Pt, 32)
    got = run_gpu(px, to_dev(tok_t, torch.int32, dev), to_dev(st_t, torch.int64, dev),
                  to_dev(ln_t, torch.int32, dev), to_dev(co_t, torch.uint8, dev), ws_total=0)
    assert np.all(got["flags"] == PX.FLAG_WS_OVERFLOW)
    assert np.all(np.isnan(got["reward"]))


def test_config_flag_and_coefficients(dev):
    log("case cfg flags")
    P = S.make_params("ragged")
    n = S.n_rows_of("ragged")
    tok_h, st_h, ln_h, co_h = S.host_batch(P, n)
    for coef_over, fl in ((dict(alpha=0.0, beta_subtask=0.1, beta_trial=0.0, rho=2.0, rho_clip=0.1), 0),
                          (dict(alpha=0.3, beta_subtask=0.025, beta_trial=0.05, rho=0.0, rho_clip=0.0),
                           PX.CFG_INVALID_KEEPS_CORRECTNESS)):
        px, coef = px_for(flags=fl, **coef_over)
        got = run_gpu(px, to_dev(tok_h, torch.int32, dev), to_dev(st_h, torch.int64, dev),
                      to_dev(ln_h, torch.int32, dev), to_dev(co_h, torch.uint8, dev))
        compare(got, *oracle_expect(tok_h, st_h, ln_h, co_h, TAGS, G, coef, fl), what="cfg %s" % fl)


def test_group_sizes(dev):
    log("case group sizes")
    P = S.make_params("tiny", groups=15)
    n = 120
    tok_h, st_h, ln_h, co_h = S.host_batch(P, n)
    for g in (1, 3, 5, 120):
        px = PX.Parason(TAGS, group_size=g, **DEFAULT_COEF)
        got = run_gpu(px, to_dev(tok_h, torch.int32, dev), to_dev(st_h, torch.int64, dev),
                      to_dev(ln_h, torch.int32, dev), to_dev(co_h, torch.uint8, dev))
        compare(got, *oracle_expect(tok_h, st_h, ln_h, co_h, TAGS, g, DEFAULT_COEF), what="G=%d" % g)


def test_repeatable(dev):
    log("case repeatable")
    P = S.make_params("small")
    n = S.n_rows_of("small")
    tok_d, st_d, ln_d, co_d = S.device_batch(P, n, device=dev)
    px, _ = px_for()
    a = run_gpu(px, tok_d, st_d, ln_d, co_d)
    b = run_gpu(px, tok_d, st_d, ln_d, co_d)
    for k in a:
        assert np.array_equal(a[k].view(np.uint32) if a[k].dtype == np.float32 else a[k],
                              b[k].view(np.uint32) if b[k].dtype == np.float32 else b[k]), k


def test_device_is_gfx950_and_accepted(dev):
    """The library's device check (every launching call returns
    PARASON_ERR_DEVICE unless the current device is gfx950) passes here."""
    log("case device check")
    arch = torch.cuda.get_device_properties(dev).gcnArchName
    assert arch.split(":")[0] == "gfx950", arch
    px, _ = px_for()
    P = S.make_params("tiny")
    tok, st, ln, co = S.device_batch(P, G, device=dev)
    out = px.alloc_outputs(G, dev)
    ws = px.alloc_workspace(G, int(tok.numel()), dev)
    rc = px.run_raw(tok.data_ptr(), st.data_ptr(), ln.data_ptr(), co.data_ptr(), G, out, ws.data_ptr(), ws.numel(),
                    torch.cuda.current_stream(dev).cuda_stream)
    assert rc == PX.OK
    torch.cuda.synchronize()


@pytest.mark.parametrize("n_elem", [0, 1, 3, 4, 515, 1 << 20, (1 << 22) + 4096 * 3 + 7])
def test_read_probe_reads_every_word(dev, n_elem):
    """The streaming-read ceiling probe reads every word once: with one sink
    word per wave, the XOR of the sink is the XOR of the buffer."""
    log("case read probe %d" % n_elem)
    rng = np.random.default_rng(n_elem)
    buf = rng.integers(-2 ** 31, 2 ** 31, size=n_elem + 8, dtype=np.int64).astype(np.int32)
    d = to_dev(buf, torch.int32, dev)
    waves = torch.cuda.get_device_properties(dev).multi_processor_count * 16
    sink = torch.zeros(waves, dtype=torch.int32, device=dev)
    rc = PX.read_probe_raw(d.data_ptr(), 4 * n_elem, sink.data_ptr(), waves, torch.cuda.current_stream(dev).cuda_stream)
    assert rc == PX.OK
    torch.cuda.synchronize()
    want = np.bitwise_xor.reduce(buf[:n_elem].view(np.uint32)) if n_elem else np.uint32(0)
    got = np.bitwise_xor.reduce(sink.cpu().numpy().view(np.uint32))
    assert got == want


def test_read_probe_dynamic_chunks_read_every_word(dev):
    """A buffer of at least 128 eight-kilobyte steps per wave takes the
    probe's counter-driven chunks after the equal shares (the scan's
    distribution): every word is still read exactly once.  The buffer holds
    0 .. N-1, whose XOR has a closed form."""
    waves = torch.cuda.get_device_properties(dev).multi_processor_count * 16
    n_elem = 128 * waves * 2048 + 2048 * 333 + 7  # whole steps, a partial one, a tail of 3 words
    log("case read probe dynamic %d" % n_elem)
    assert n_elem < 2 ** 31
    d = torch.arange(n_elem, dtype=torch.int32, device=dev)
    sink = torch.zeros(waves, dtype=torch.int32, device=dev)
    for _ in range(2):  # the counter is cleared for every call
        sink.zero_()
        rc = PX.read_probe_raw(d.data_ptr(), 4 * n_elem, sink.data_ptr(), waves,
                               torch.cuda.current_stream(dev).cuda_stream)
        assert rc == PX.OK
        torch.cuda.synchronize()
        m = n_elem - 1
        want = [m, 1, m + 1, 0][m % 4]  # XOR of 0 .. m
        got = int(np.bitwise_xor.reduce(sink.cpu().numpy().view(np.uint32)))
        assert got == want
    del d
