"""The opt-in finite check of the step (muonbp_options.check_finite), and
the device-memory budget of muonbp_create (muonbp_options.device_memory_limit).

With the check on, a NaN or an Inf in a gradient (hence in the momentum that
Alg. 2 normalises) makes muonbp_step return MUONBP_E_NONFINITE before any
orthogonalization or update is enqueued: the params keep their values, and
the context stays usable once the caller restores the momentum.  With the
check off (the default) the non-finite value propagates silently, through
the unit's Frobenius norm, into U and the params of its unit only.
"""

import ctypes

import numpy as np
import pytest

from tests.gpu_harness import announce

pytestmark = pytest.mark.gpu

MATS = [(64, 128, 1, 2), (96, 64, 1, 1)]


@pytest.fixture(scope="module", autouse=True)
def gpu():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a ROCm device"
    from paper_2510_16981_amd import muonbp as mb
    mb.load_library()


def _tensors(seed):
    import torch
    rng = np.random.default_rng(seed)
    p = [torch.from_numpy(0.02 * rng.standard_normal((r, c))).to(torch.bfloat16).cuda()
         for r, c, _, _ in MATS]
    g = [[torch.from_numpy(0.01 * rng.standard_normal((r, c))).to(torch.bfloat16).cuda()
          for r, c, _, _ in MATS] for _ in range(3)]
    return p, g


def _raw_step(ctx, params, grads, t):
    n = len(params)
    pp = (ctypes.c_void_p * n)(*[p.data_ptr() for p in params])
    gp = (ctypes.c_void_p * n)(*[g.data_ptr() for g in grads])
    return ctx.lib.muonbp_step(ctx.ctx, pp, gp, t)


@pytest.mark.parametrize("bad", [float("nan"), float("inf")], ids=["nan", "inf"])
def test_check_on_reports_nonfinite_and_leaves_params(bad):
    import torch
    from paper_2510_16981_amd import muonbp as mb
    announce(f"check_finite on, {bad} gradient")
    opts = mb.options_default(check_finite=1)
    A = mb.MuonBP(MATS, 2, 0.01, 0.02, 0.95, 0.1, options=opts)
    B = mb.MuonBP(MATS, 2, 0.01, 0.02, 0.95, 0.1, options=opts)
    p0, g = _tensors(3)
    pA = [p.clone() for p in p0]
    pB = [p.clone() for p in p0]
    A.step(pA, g[0], 0)
    B.step(pB, g[0], 0)
    torch.cuda.synchronize()
    saved = [A.get_momentum(i).clone() for i in range(len(MATS))]
    before = [p.clone() for p in pA]
    gbad = [x.clone() for x in g[1]]
    gbad[0][5, 70] = bad  # block (0, 1) of matrix 0
    torch.cuda.synchronize()
    st = _raw_step(A, pA, gbad, 1)
    assert mb.STATUS[st] == "MUONBP_E_NONFINITE", st
    torch.cuda.synchronize()
    for x, y in zip(pA, before):
        assert torch.equal(x, y)  # nothing after the momentum ran
    # Usable again once the momentum (updated by the failed step, also for
    # the finite matrix) is restored; then identical to a context that never
    # saw the bad gradient.
    for i, m in enumerate(saved):
        A.set_momentum(i, m)
    A.step(pA, g[1], 1)
    B.step(pB, g[1], 1)
    A.step(pA, g[2], 2)
    B.step(pB, g[2], 2)
    torch.cuda.synchronize()
    for x, y in zip(pA, pB):
        assert torch.equal(x, y)
    for i in range(len(MATS)):
        assert torch.equal(A.get_momentum(i), B.get_momentum(i))
    A.close()
    B.close()


def test_check_off_propagates_into_its_unit_only():
    import torch
    from paper_2510_16981_amd import muonbp as mb
    announce("check_finite off, NaN gradient")
    A = mb.MuonBP(MATS, 0, 0.01, 0.02, 0.95, 0.1)  # P = infinity: block steps only
    p, g = _tensors(5)
    gbad = [x.clone() for x in g[0]]
    gbad[0][5, 70] = float("nan")  # block (0, 1) of matrix 0 (columns 64..127)
    A.step(p, gbad, 0)
    torch.cuda.synchronize()
    U = A.get_update(0).float()
    torch.cuda.synchronize()
    assert torch.isnan(U[:, 64:]).all()
    assert torch.isfinite(U[:, :64]).all()
    assert torch.isnan(p[0][:, 64:].float()).all()
    assert torch.isfinite(p[0][:, :64].float()).all()
    assert torch.isfinite(p[1].float()).all()
    A.close()


def test_device_memory_limit_out_of_memory_frees_everything():
    """A budget just above the momentum + workspace + split sums passes the
    up-front check and runs out on the descriptor tables: E_NOMEM, and every
    allocation made so far is freed (the free device memory is the same
    after 20 such failures).  A budget with room for the tables works."""
    import torch
    from paper_2510_16981_amd import muonbp as mb
    mats = [(2048, 6144, 1, 8)]
    bulk = mb.describe_plan(mats, True).device_bytes
    announce(f"device_memory_limit around {bulk} bytes")
    lib = mb.load_library()

    def create(limit):
        ctx = ctypes.c_void_p()
        o = mb.options_default(device_memory_limit=limit)
        st = lib.muonbp_create(mb._mats(mats), len(mats), 5, 0.01, 0.02, 0.95, 0.1, ctypes.byref(o),
                               ctypes.c_void_p(torch.cuda.current_stream().cuda_stream),
                               ctypes.byref(ctx))
        return st, ctx

    torch.cuda.synchronize()
    st, ctx = create(bulk + 1024)
    assert st == 4 and not ctx.value
    free0 = torch.cuda.mem_get_info()[0]
    for _ in range(20):
        st, ctx = create(bulk + 1024)
        assert st == 4 and not ctx.value
    assert torch.cuda.mem_get_info()[0] == free0
    st, ctx = create(bulk + (64 << 20))
    assert st == 0 and ctx.value
    lib.muonbp_destroy(ctx)
