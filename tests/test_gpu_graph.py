"""Every entry point inside a captured HIP graph.

No call allocates, synchronises or records a memset, so a caller can capture
them (a serving loop captures the decode step with the model's forward pass).
Each test captures a call sequence once, then replays the graph several
times with the program's own eager work and synchronisations between the
replays (outputs overwritten with garbage, a different kernel on the stream),
and checks every replay bit for bit against the same calls made eagerly."""
import numpy as np
import pytest

from gpu_util import log, to_dev
from paper_2608_24658_amd import parason as PX
from paper_2608_24658_amd.synth import synth as S

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

REPLAYS = 4


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch.device("cuda:0")


def replay_and_check(graph, outputs, expected, scramble):
    for k in range(REPLAYS):
        for t in outputs:
            scramble(t)
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for name, t, e in zip(range(len(outputs)), outputs, expected):
            assert torch.equal(t.view(torch.uint8), e.view(torch.uint8)), (k, name)


def garbage(t):
    t.view(torch.uint8).fill_(0xA5)


def test_graph_accounting(dev):
    log("case graph accounting")
    P = S.make_params("small")
    n = S.n_rows_of("small")
    tok, st, ln, co = S.device_batch(P, n, device=dev)
    px = PX.Parason(S.CONTIGUOUS_TAGS, group_size=S.GROUP_SIZE)
    out = px.alloc_outputs(n, dev, metrics=True)
    ws = px.alloc_workspace(n, tok.numel(), dev)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):
        px.run(tok, st, ln, co, out=out, workspace=ws, metrics=True)
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    keys = sorted(out)
    expected = [out[k].clone() for k in keys]
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        px.run(tok, st, ln, co, out=out, workspace=ws, metrics=True)
    replay_and_check(g, [out[k] for k in keys], expected, garbage)


def test_graph_policy_gradient(dev):
    log("case graph pg")
    P = S.make_params("small")
    n = S.n_rows_of("small")
    lengths, _ = S.host_rows(P, n)
    starts = np.zeros(n, np.int64)
    starts[1:] = np.cumsum(lengths[:-1].astype(np.int64))
    N = int(lengths.astype(np.int64).sum())
    old, new = S.device_logp(P, N, device=dev)
    reward = to_dev(np.random.default_rng(1).choice([-1.0, 1.0, 1.25], n).astype(np.float32), torch.float32, dev)
    st_d, ln_d = to_dev(starts, torch.int64, dev), to_dev(lengths, torch.int32, dev)
    grad = torch.empty_like(new)
    ws = torch.empty(PX.pg_workspace_size(n), dtype=torch.uint8, device=dev)
    res = PX.pg_run(reward, new, old, st_d, ln_d, grad=grad, workspace=ws)
    torch.cuda.synchronize()
    expected = [res["advantage"].clone(), grad.clone(), res["stats"].clone()]
    g = torch.cuda.CUDAGraph()
    holder = {}
    with torch.cuda.graph(g):
        holder.update(PX.pg_run(reward, new, old, st_d, ln_d, grad=grad, workspace=ws))
    replay_and_check(g, [holder["advantage"], grad, holder["stats"]], expected, garbage)


def test_graph_decode_steps(dev):
    """Eight decode steps captured as one graph (states advance in place, so
    each replay starts from freshly initialised states)."""
    log("case graph decode")
    B, V, steps = 64, 4096, 8
    tags = [V - 12 + k for k in range(12)]
    px = PX.Parason(tags)
    rng = np.random.default_rng(2)
    seq = [tags[0], tags[2], tags[4], tags[6], 7, tags[7], tags[5], tags[10]]
    toks = [to_dev(np.array([seq[k] if r % 3 else int(rng.integers(0, 4000)) for r in range(B)], np.int32),
                   torch.int32, dev) for k in range(steps)]
    logits0 = torch.randn(B, V, device=dev)
    states = torch.empty(B * PX.DECODE_STATE_BYTES, dtype=torch.uint8, device=dev)
    logits = torch.empty_like(logits0)

    def run():
        PX.decode_init(B, dev, states=states)
        logits.copy_(logits0)
        px.decode_step(states, logits, None, 4000)
        for k in range(steps - 1):
            px.decode_step(states, logits, toks[k], 4000)

    run()
    torch.cuda.synchronize()
    expected = [states.clone(), logits.clone()]
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        run()
    replay_and_check(g, [states, logits], expected, garbage)


def test_graph_fork_join(dev):
    """Fork and join with capacities given (the sizing call synchronises and
    stays outside the graph)."""
    log("case graph fork/join")
    tags = [int(t) for t in S.CONTIGUOUS_TAGS]
    P = S.make_params("small")
    tok_h, st_h, ln_h, _ = S.host_batch(P, 64)
    end_out = tags[5]
    cut = np.array([int(np.nonzero(tok_h[s: s + l] == end_out)[0][0]) + 1 if (tok_h[s: s + l] == end_out).any()
                    else l for s, l in zip(st_h, ln_h)], np.int32)
    tok, st, ln = to_dev(tok_h, torch.int32, dev), to_dev(st_h, torch.int64, dev), to_dev(cut, torch.int32, dev)
    px = PX.Parason(tags)
    first = px.fork(tok, st, ln)
    W, T, _ = (int(x) for x in first["totals"].cpu())
    wl = first["ctx_lengths"].to(torch.int64) + 3
    wst = torch.zeros(W, dtype=torch.int64, device=dev)
    wst[1:] = torch.cumsum(wl, 0)[:-1]
    wtok = torch.full((int(wl.sum().item()),), 9, dtype=torch.int32, device=dev)
    # each worker sequence: its context, two filler tokens, </Thread>
    cl = first["ctx_lengths"].to(torch.int64)
    idx = torch.repeat_interleave(torch.arange(W, device=dev), cl)
    within = torch.arange(idx.numel(), device=dev) - torch.repeat_interleave(torch.cumsum(cl, 0) - cl, cl)
    wtok[wst[idx] + within] = first["ctx_tokens"][first["ctx_starts"][idx] + within]
    wtok[wst + wl - 1] = tags[11]
    wl32 = wl.to(torch.int32)
    jfirst = px.join(tok, st, ln, first["worker_off"], wtok, wst, wl32)
    JT = int(jfirst["totals"][0].item())
    torch.cuda.synchronize()
    holder = {}

    def run():
        holder["f"] = px.fork(tok, st, ln, max_workers=W, ctx_capacity=T)
        holder["j"] = px.join(tok, st, ln, holder["f"]["worker_off"], wtok, wst, wl32, capacity=JT)

    run()
    torch.cuda.synchronize()
    fk = ("ctx_tokens", "ctx_starts", "ctx_lengths", "ctx_row", "worker_off", "row_status", "totals")
    jk = ("tokens", "starts", "lengths", "row_status", "totals")
    expected = [holder["f"][k].clone() for k in fk] + [holder["j"][k].clone() for k in jk]
    assert torch.equal(expected[0], first["ctx_tokens"])
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        run()
    replay_and_check(g, [holder["f"][k] for k in fk] + [holder["j"][k] for k in jk], expected, garbage)
