"""GPU parity of the grammar-constrained decode step against the CPU oracle.

Each case runs a batch of seeded random rollouts: at every step the GPU
advances its per-sequence states by the tokens sampled last and masks a fresh
block of random logits; the oracle gives, for every sequence's prefix, the
allowed next classes and whether end of sequence is allowed.  The masked
logits must equal, bit for bit, the input with -inf written exactly at the
forbidden ids (Text = every id that is neither a tag nor the end-of-sequence
id); padding columns between rows must be untouched, and the per-sequence
error/done flags must match.  Tokens are then sampled from the oracle's
allowed sets (some sequences sample a forbidden token on purpose, some skip a
step with a negative token)."""
import random

import numpy as np
import pytest

from gpu_util import log
from oracle import decode_oracle as D
from paper_2608_24658_amd import parason as PX
from paper_2608_24658_amd.synth import synth as S

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

CONTIG = list(S.CONTIGUOUS_TAGS)
TORCH_DT = {"f32": torch.float32, "bf16": torch.bfloat16, "f16": torch.float16}
INT_VIEW = {"f32": torch.int32, "bf16": torch.int16, "f16": torch.int16}
# classes in the order a rollout that wants to nest deeper prefers them:
# <Parallel> <Outlines> </Outlines> <Thread> </Subtask> </Trial> <Subtask> <Trial>
DEEPER = (3, 5, 6, 11, 8, 10, 7, 9)


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch.device("cuda:0")


def scattered_tags(V, seed):
    rng = np.random.default_rng(seed)
    return [int(t) for t in rng.choice(V, size=12, replace=False)]


def expected_mask(allowed, eos_ok, tags, eos, V):
    """Boolean [V] of the ids the decoder must set to -inf."""
    m = np.zeros(V, dtype=bool)
    if 0 not in allowed:  # no Text: everything but the allowed tags
        m[:] = True
        for c in allowed:
            m[tags[c - 1]] = False
        return m
    for c in range(1, 13):
        if c not in allowed:
            m[tags[c - 1]] = True
    if eos >= 0 and not eos_ok:
        m[eos] = True
    return m


def simulate(dev, *, B, steps, V, tags, eos, dtype, seed, pad=0, p_bad=0.0, p_skip=0.0, p_deep=0.0,
             p_end=0.03, max_depth=1 << 30, cfg_flags=0):
    """Run `steps` decode steps on B sequences; returns counters for coverage checks.
    cfg_flags: the handle's configuration flags (PX.CFG_LENIENT_GAPS selects the
    lenient language on both sides)."""
    rng = random.Random(seed)
    gen = torch.Generator().manual_seed(seed)
    px = PX.Parason(tags, flags=cfg_flags)
    tag_set = set(tags)
    text_pool = [t for t in range(min(V, 4096)) if t not in tag_set and t != eos]
    states = PX.decode_init(B, dev)
    prefixes = [[] for _ in range(B)]
    flags = [0] * B
    depth = [0] * B
    tokens = None
    seen = dict(full_rows=0, text_rows=0, errors=0, done=0, skips=0, max_depth=0)
    for step in range(steps):
        full = torch.randn(B, V + pad, generator=gen).to(TORCH_DT[dtype])
        logits = full.to(dev, copy=True)
        view = logits[:, :V] if pad else logits
        px.decode_step(states, view, tokens, eos)
        got = logits.cpu()
        st = PX.decode_fields(states).cpu().numpy()
        live = [i for i in range(B) if flags[i] == 0]
        allowed = dict(zip(live, D.allowed_batch([prefixes[i] for i in live], tags, text_pool[0], cfg_flags)))
        exp = full.clone()
        for i in range(B):
            if flags[i]:
                continue
            a, eos_ok = allowed[i]
            m = torch.from_numpy(expected_mask(a, eos_ok, tags, eos, V))
            exp[i, :V][m] = float("-inf")
            seen["full_rows" if 0 not in a else "text_rows"] += 1
            # Text allowed between a region's structural tags (lenient gaps)
            seen["gap_rows"] = seen.get("gap_rows", 0) + (0 in a and 3 not in a and bool(a & {5, 7, 9, 11}))
        iv = INT_VIEW[dtype]
        if not torch.equal(got.view(iv), exp.view(iv)):
            bad = (got.view(iv) != exp.view(iv)).nonzero()
            r, c = int(bad[0, 0]), int(bad[0, 1])
            raise AssertionError("step %d: %d logits differ, first row %d id %d (gpu %r expected %r) prefix %s" % (
                step, bad.shape[0], r, c, float(got[r, c]), float(exp[r, c]), prefixes[r][-8:]))
        assert list(st[:, 3]) == flags, (step, list(st[:, 3]), flags)
        # sample the next tokens
        nxt = []
        for i in range(B):
            if flags[i]:
                nxt.append(rng.choice(text_pool))  # ignored by the decoder from now on
                continue
            a, eos_ok = allowed[i]
            if rng.random() < p_skip:
                nxt.append(-1)
                seen["skips"] += 1
                continue
            if rng.random() < p_bad:
                bad = sorted(set(range(13)) - a)
                if bad:
                    c = rng.choice(bad)
                    nxt.append(rng.choice(text_pool) if c == 0 else tags[c - 1])
                    prefixes[i].append(nxt[-1])
                    flags[i] = PX.DECODE_ERROR
                    seen["errors"] += 1
                    continue
            if eos_ok and eos >= 0 and rng.random() < 0.2:
                nxt.append(eos)
                flags[i] = PX.DECODE_DONE
                seen["done"] += 1
                continue
            if 2 in a and rng.random() >= p_end:
                a = a - {2}  # keep most rollouts inside <think> for a while
            tags_ok = sorted(a - {0})
            deeper = [c for c in DEEPER if c in a]
            if deeper and depth[i] < max_depth and rng.random() < p_deep:
                c = deeper[0]
            elif tags_ok and rng.random() < 0.6:
                c = rng.choice(tags_ok)
            else:
                c = rng.choice(sorted(a))
            depth[i] += 1 if c == 3 else (-1 if c == 4 else 0)
            seen["max_depth"] = max(seen["max_depth"], depth[i])
            tok = rng.choice(text_pool) if c == 0 else tags[c - 1]
            nxt.append(tok)
            prefixes[i].append(tok)
        tokens = torch.tensor(nxt, dtype=torch.int32, device=dev)
    torch.cuda.synchronize()
    return seen


def test_decode_contiguous_f32(dev):
    log("case decode contiguous f32 V=4096 B=64")
    seen = simulate(dev, B=64, steps=160, V=4096, tags=[4096 - 12 + k for k in range(12)], eos=4000,
                    dtype="f32", seed=1, p_bad=0.01, p_skip=0.05)
    assert seen["full_rows"] > 500 and seen["text_rows"] > 500 and seen["errors"] > 0 and seen["done"] > 0


def test_decode_scattered_bf16_padded(dev):
    log("case decode scattered bf16 V=3001 pad 5 B=48")
    V = 3001
    seen = simulate(dev, B=48, steps=120, V=V, tags=scattered_tags(V, 3), eos=17, dtype="bf16", seed=2,
                    pad=5, p_bad=0.01)
    assert seen["full_rows"] > 300 and seen["errors"] > 0


def test_decode_f16_misaligned_rows(dev):
    # rows of 1003 + 2 halves: every row starts at a different offset mod 16 bytes
    log("case decode f16 V=1003 pad 2 B=40")
    V = 1003
    seen = simulate(dev, B=40, steps=100, V=V, tags=scattered_tags(V, 5), eos=V - 1, dtype="f16", seed=3, pad=2)
    assert seen["full_rows"] > 200


def test_decode_no_eos(dev):
    log("case decode no eos V=512 B=32")
    seen = simulate(dev, B=32, steps=120, V=512, tags=scattered_tags(512, 7), eos=-1, dtype="f32", seed=4)
    assert seen["done"] == 0


def test_decode_deep_nesting(dev):
    log("case decode deep nesting V=2048 B=16")
    seen = simulate(dev, B=16, steps=300, V=2048, tags=scattered_tags(2048, 9), eos=5, dtype="bf16", seed=5,
                    p_deep=0.9, max_depth=60)
    assert seen["max_depth"] >= 25


def test_decode_full_vocabulary(dev):
    log("case decode V=151936 bf16 B=16 contiguous tags")
    seen = simulate(dev, B=16, steps=40, V=S.VOCAB, tags=CONTIG, eos=151643, dtype="bf16", seed=6,
                    p_bad=0.02)
    assert seen["full_rows"] > 50


def test_decode_grid_stride(dev):
    # more sequences than the launch has blocks: the kernel strides over rows
    log("case decode B=5000 V=96 f32")
    seen = simulate(dev, B=5000, steps=12, V=96, tags=scattered_tags(96, 11), eos=0, dtype="f32", seed=7,
                    p_bad=0.01)
    assert seen["full_rows"] > 5000


def test_decode_state_fields(dev):
    # depth counts the open <Parallel> blocks; a forbidden token sets the error flag
    log("case decode state fields")
    V = 64
    tags = list(range(40, 52))
    px = PX.Parason(tags)
    st = PX.decode_init(1, dev)
    logits = torch.zeros(1, V, device=dev)
    seq = [tags[0], tags[2], tags[4], tags[6], 3, tags[7], tags[5], tags[10], tags[2], tags[4]]
    depths = []
    for t in [None] + seq:
        px.decode_step(st, logits, None if t is None else torch.tensor([t], dtype=torch.int32, device=dev), -1)
        depths.append(int(PX.decode_fields(st)[0, 1].item()))
    assert depths == [0, 0, 1, 1, 1, 1, 1, 1, 1, 2, 2]
    assert int(PX.decode_fields(st)[0, 3].item()) == 0
    px.decode_step(st, logits, torch.tensor([tags[1]], dtype=torch.int32, device=dev), -1)  # </think> after <Outlines>
    assert int(PX.decode_fields(st)[0, 3].item()) == PX.DECODE_ERROR


def test_decode_lenient_gaps(dev):
    """Text allowed between the structural tags of a region: the masks follow
    the lenient language, the rows that used to be rewritten whole now keep
    their Text logits."""
    log("case decode lenient V=2048 bf16 B=64")
    seen = simulate(dev, B=64, steps=200, V=2048, tags=scattered_tags(2048, 13), eos=9, dtype="bf16", seed=8,
                    p_bad=0.01, p_deep=0.3, max_depth=8, cfg_flags=PX.CFG_LENIENT_GAPS)
    assert seen["text_rows"] > 5000 and seen["errors"] > 0 and seen["gap_rows"] > 500
    # only the start of a stream forbids Text in the lenient language
    assert seen["full_rows"] == 64


def test_decode_lenient_full_vocabulary(dev):
    log("case decode lenient V=151936 f32 B=8 contiguous tags")
    seen = simulate(dev, B=8, steps=60, V=S.VOCAB, tags=CONTIG, eos=151643, dtype="f32", seed=9, p_bad=0.02,
                    cfg_flags=PX.CFG_LENIENT_GAPS)
    assert seen["text_rows"] > 200
