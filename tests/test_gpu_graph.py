"""HIP-graph capture of the optimizer step (GPU).

A block step captured on the context's stream is replayed several times,
with eager work (new gradient values written in place) and synchronisations
between the replays.  After every replay, the params and the momentum must
equal, bit for bit, those of a second context that runs the same steps
eagerly.  A capture whose pointers differ from the previous step's is
refused with E_STATE before anything is enqueued, and the context stays
usable.
"""

import numpy as np
import pytest

from tests.gpu_harness import announce

pytestmark = pytest.mark.gpu

# A unit with more rows than columns (transposed NS, U written as Z^T) and
# one with ragged tiles; P = 5, so steps 1..4 are block steps.
MATS = [(264, 1040, 1, 2), (1040, 264, 2, 1)]
PERIOD = 5


@pytest.fixture(scope="module", autouse=True)
def gpu():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a ROCm device"
    from paper_2510_16981_amd import muonbp as mb
    mb.load_library()


def _setup():
    import torch
    from paper_2510_16981_amd import muonbp as mb
    rng = np.random.default_rng(7)
    p0 = [torch.from_numpy(0.02 * rng.standard_normal((r, c))).to(torch.bfloat16).cuda()
          for r, c, _, _ in MATS]
    g = [torch.from_numpy(0.01 * rng.standard_normal((r, c))).to(torch.bfloat16).cuda()
         for r, c, _, _ in MATS]
    ctxs = []
    for _ in range(2):
        s = torch.cuda.Stream()
        ctxs.append((mb.MuonBP(MATS, PERIOD, 0.01, 0.02, 0.95, 0.1,
                               options=mb.options_default(), stream=s), s,
                     [p.clone() for p in p0]))
    return ctxs, g


def _same_state(a, pa, b, pb):
    import torch
    torch.cuda.synchronize()
    for x, y in zip(pa, pb):
        assert torch.equal(x, y)
    for i in range(len(MATS)):
        ma, mb_ = a.get_momentum(i), b.get_momentum(i)
        torch.cuda.synchronize()
        assert torch.equal(ma, mb_)


def test_captured_block_step_replays_like_eager_steps():
    import torch
    ((A, sA, pA), (B, _, pB)), g = _setup()
    for t in (0, 1):  # a full and a block step; the pointer table is now current
        A.step(pA, g, t)
        B.step(pB, g, t)
    _same_state(A, pA, B, pB)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=sA):
        A.step(pA, g, 2)
    torch.cuda.synchronize()
    _same_state(A, pA, B, pB)  # capturing ran nothing
    for r in range(3):
        announce(f"graph replay {r}")
        for gi in g:  # eager work between the replays
            gi.mul_(0.5).add_(0.001)
        torch.cuda.synchronize()
        graph.replay()
        B.step(pB, g, 2 + r)
        _same_state(A, pA, B, pB)
    A.close()
    B.close()


def test_capture_with_new_pointers_is_refused():
    import torch
    from paper_2510_16981_amd import muonbp as mb
    ((A, sA, pA), (B, _, pB)), g = _setup()
    for t in (0, 1):
        A.step(pA, g, t)
        B.step(pB, g, t)
    torch.cuda.synchronize()
    fresh = [p.clone() for p in pA]
    graph = torch.cuda.CUDAGraph()
    with pytest.raises(mb.MuonBPError) as err:
        with torch.cuda.graph(graph, stream=sA):
            A.step(fresh, g, 2)
    assert mb.STATUS[err.value.status] == "MUONBP_E_STATE"
    del graph
    torch.cuda.synchronize()
    # The context is unharmed: the next eager step matches the other context.
    A.step(pA, g, 2)
    B.step(pB, g, 2)
    _same_state(A, pA, B, pB)
    A.close()
    B.close()


def test_replay_after_many_eager_steps_with_other_pointers():
    """The captured step's pointer table is never overwritten: after more
    eager steps with other pointers than the table has slots (alternating
    between two other sets of tensors), a replay still updates the captured
    tensors with the captured gradients.  Context B runs the same sequence
    eagerly (the replay's place taken by an eager step with the captured
    tensors); every tensor and the momentum agree bit for bit."""
    import torch
    ((A, sA, pA), (B, _, pB)), g = _setup()
    rng = np.random.default_rng(11)
    others = []
    for _ in range(2):
        po = [torch.from_numpy(0.02 * rng.standard_normal((r, c))).to(torch.bfloat16).cuda()
              for r, c, _, _ in MATS]
        go = [torch.from_numpy(0.01 * rng.standard_normal((r, c))).to(torch.bfloat16).cuda()
              for r, c, _, _ in MATS]
        others.append(([p.clone() for p in po], [p.clone() for p in po], go))
    for t in (0, 1):
        A.step(pA, g, t)
        B.step(pB, g, t)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=sA):
        A.step(pA, g, 2)
    torch.cuda.synchronize()
    for r in range(2):
        for i in range(9):  # more pointer changes than the initial slot count
            pa_o, pb_o, go = others[i % 2]
            A.step(pa_o, go, 3 + i)
            B.step(pb_o, go, 3 + i)
        torch.cuda.synchronize()
        announce(f"replay after 9 eager steps with other pointers, round {r}")
        graph.replay()
        B.step(pB, g, 2)
        _same_state(A, pA, B, pB)
        for pa_o, pb_o, _ in others:
            for x, y in zip(pa_o, pb_o):
                assert torch.equal(x, y)
    A.close()
    B.close()
