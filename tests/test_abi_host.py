"""Host-side checks of the C-ABI library (no GPU needed, no compute call).

The library must load, export every function declared in include/muonbp.h,
reject bad arguments before touching the GPU, and describe its plans.
"""

import ctypes
import os
import re

import numpy as np
import pytest

from oracle import muonbp_oracle as O
from paper_2510_16981_amd import muonbp as mb
from paper_2510_16981_amd import workload as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "muonbp.h")


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(mb.LIB_PATH):
        from paper_2510_16981_amd import build
        build.build()
    return mb.load_library()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(muonbp_[a-z_]+)\s*\(", text)))


def test_header_declares_the_api():
    names = declared_functions()
    for required in ["muonbp_create", "muonbp_step", "muonbp_destroy",
                     "muonbp_get_update", "muonbp_get_momentum", "muonbp_set_momentum"]:
        assert required in names


def test_library_exports_every_declared_symbol(lib):
    missing = [n for n in declared_functions() if not hasattr(lib, n)]
    assert not missing, missing


def test_options_default(lib):
    o = mb.options_default()
    assert o.ns_steps == 5
    assert (o.a, o.b, o.c) == (2.0, -1.5, 0.5)
    assert abs(o.eps - 1e-7) < 1e-12
    assert (o.nesterov, o.scale_mode, o.rms_beta) == (0, 0, 1.0)
    assert (o.param_dtype, o.state_dtype, o.ns_dtype) == (mb.BF16, mb.BF16, mb.BF16)
    assert (o.tile_policy, o.k_split, o.coeff_count) == (0, 0, 0)
    t = mb.options_default(coeffs=[(3.0, -3.2, 1.2), (2.0, -1.5, 0.5)])
    assert t.coeff_count == 2 and list(t.coeff_table[:6]) == pytest.approx([3.0, -3.2, 1.2, 2.0, -1.5, 0.5])


def test_status_strings(lib):
    texts = [lib.muonbp_status_string(code) for code in range(9)]
    assert all(texts) and b"unknown status" not in texts and len(set(texts)) == 9
    assert lib.muonbp_status_string(99) == b"unknown status"
    assert lib.muonbp_last_error(None) == b"no context"
    lib.muonbp_destroy(None)  # NULL-safe


def _create(lib, mats, period=5, opt=None, out=True):
    ctx = ctypes.c_void_p()
    arr = mb._mats(mats) if mats is not None else None
    n = len(mats) if mats is not None else 0
    return lib.muonbp_create(arr, n, period, 0.01, 0.02, 0.95, 0.1,
                             ctypes.byref(opt) if opt else None, None,
                             ctypes.byref(ctx) if out else None), ctx


def test_device_memory_limit_refuses_before_gpu(lib):
    """A budget below the momentum + workspace + split sums fails with
    E_NOMEM before any HIP call (this container has no GPU, so reaching one
    would give E_HIP); a negative budget is an invalid option."""
    mats = W.workload_matrices("qkv-2048x6144-bf16")
    info = mb.describe_plan(mats, True)
    full_ws = info.workspace_bytes
    assert info.device_bytes >= 2048 * 6144 * 2 + full_ws
    assert mb.describe_plan(mats, False).device_bytes == info.device_bytes
    for limit in (1, 2048 * 6144 * 2, info.device_bytes - 1):
        st, ctx = _create(lib, mats, opt=mb.options_default(device_memory_limit=limit))
        assert st == 4 and not ctx.value
    assert _create(lib, mats, opt=mb.options_default(device_memory_limit=-1))[0] == 1


def test_create_rejects_bad_arguments_before_gpu(lib):
    assert _create(lib, None)[0] == 1
    assert _create(lib, [])[0] == 1
    assert _create(lib, [(8, 8, 1, 1)], out=False)[0] == 1
    assert _create(lib, [(8, 8, 1, 1)], period=-1)[0] == 1
    st, ctx = _create(lib, [(10, 8, 3, 1)])
    assert st == 2 and not ctx.value
    assert _create(lib, [(0, 8, 1, 1)])[0] == 2
    assert _create(lib, [(8, 8, 0, 1)])[0] == 2
    assert _create(lib, [(8, 8, 1, 1)], opt=mb.options_default(param_dtype=7))[0] == 3
    assert _create(lib, [(8, 8, 1, 1)], opt=mb.options_default(ns_steps=-1))[0] == 1
    assert _create(lib, [(8, 8, 1, 1)], opt=mb.options_default(scale_mode=3))[0] == 1
    assert _create(lib, [(8, 8, 1, 1)], opt=mb.options_default(k_split=9))[0] == 1
    assert _create(lib, [(8, 8, 1, 1)], opt=mb.options_default(coeff_count=17))[0] == 1
    bad = mb.options_default(coeffs=[(2.0, -1.5, 0.5)])
    bad.coeff_table[1] = float("nan")
    assert _create(lib, [(8, 8, 1, 1)], opt=bad)[0] == 1
    assert _create(lib, [(8, 8, 1, 1)], opt=mb.options_default(tile_policy=17))[0] == 1
    assert _create(lib, [(8, 8, 1, 1)], opt=mb.options_default(stream_hint=3))[0] == 1
    assert _create(lib, [(8, 8, 1, 1)], opt=mb.options_default(stream_hint=-1))[0] == 1
    assert _create(lib, [(8, 8, 1, 1)], opt=mb.options_default(apply_mode=2))[0] == 1
    assert _create(lib, [(8, 8, 1, 1)], opt=mb.options_default(check_finite=2))[0] == 1


def _describe_status(lib, mats, opt=None, full=0):
    info = mb.PlanInfo()
    return lib.muonbp_describe_plan(mb._mats(mats), len(mats), ctypes.byref(opt) if opt else None,
                                    full, ctypes.byref(info))


@pytest.mark.parametrize("mats,ns_dtype", [
    ([(4096, 600000, 1, 1)], mb.BF16),      # 4.9 GB operand (full plan and its one block)
    ([(40000, 40000, 1, 1)], mb.BF16),      # 3.2 GB
    ([(40000, 40000, 8, 8)], mb.BF16),      # blocks are small, the full matrix is not
    ([(16384, 32768, 1, 1)], mb.F32),       # exactly 2^31 bytes in fp32
    ([(64, 64, 1, 1), (4096, 600000, 1, 8)], mb.BF16),
])
def test_units_with_operands_of_2_31_bytes_are_rejected(lib, mats, ns_dtype):
    """The NS kernels address an operand with 32-bit byte offsets: any unit of
    either plan whose Z, Z^T, A or B reaches 2^31 bytes is refused with
    E_SHAPE (no HIP call is made by describe_plan or before it in create)."""
    opt = mb.options_default(ns_dtype=ns_dtype, param_dtype=ns_dtype, state_dtype=ns_dtype)
    for full in (0, 1):
        assert _describe_status(lib, mats, opt, full) == 2
    st, ctx = _create(lib, mats, opt=opt)
    assert st == 2 and not ctx.value


def test_largest_accepted_units_stay_below_2_31_bytes(lib):
    # A 32768 x 32768 bf16 Z is exactly 2^31 bytes; one 8-element padding
    # step smaller is accepted.
    assert _describe_status(lib, [(32760, 32760, 1, 1)]) == 0
    assert _describe_status(lib, [(32768, 32768, 1, 1)]) == 2


def test_null_context_calls(lib):
    assert lib.muonbp_step(None, None, None, 0) == 1
    assert lib.muonbp_set_lr(None, 0.1, 0.1) == 1
    assert lib.muonbp_set_period(None, 3) == 1
    assert lib.muonbp_synchronize(None) == 1
    assert lib.muonbp_get_update(None, 0, None) == 1


def _unit_counts(mats, full):
    units = []
    for r, c, gr, gc in mats:
        if full:
            units.append((r, c))
        else:
            units += [(r // gr, c // gc)] * (gr * gc)
    return units


@pytest.mark.parametrize("name", list(W.WORKLOADS))
def test_describe_plan_counts_and_flops(lib, name):
    mats = W.workload_matrices(name)
    for full in (False, True):
        info = mb.describe_plan(mats, full)
        units = _unit_counts(mats, full)
        assert info.n_problems == len(units)
        assert info.n_elements == sum(r * c for r, c, _, _ in mats)
        dense = sum(O.ns_dense_flops(p, q, 5) for p, q in units)
        assert abs(info.ns_dense_flops - dense) <= 1e-9 * dense
        sym = 0.0
        gram = poly = apply = 0
        (gr_, pr_, ar_), (gc_, pc_, ac_) = info.gemm_tile_rows, info.gemm_tile_cols
        assert gr_ == gc_ and pr_ == pc_  # symmetric products use square tiles
        n_gram = 0
        for p, q in units:
            S, L = min(p, q), max(p, q)
            # Gram-space iteration (bf16, row-major apply, K = 5): S >= 128
            # and L >= 1.25 S.  Segments of 3 and 2 iterations, each one
            # Gram, 4n - 3 symmetric S x S x S products and one apply,
            # instead of K of each of three.
            g = bool(info.apply_nn) and S >= 128 and 4 * L >= 5 * S
            n_gram += g
            zz, ss, ap = S * (S + 1) * L, S * S * (S + 1), 2 * S * S * L
            sym += (2 * zz + (9 + 5) * ss + 2 * ap) if g else 5 * (zz + ss + ap)
            tg, tp = -(-S // gr_), -(-S // pr_)
            gram += tg * (tg + 1) // 2
            poly += tp * (tp + 1) // 2
            apply += -(-S // ar_) * -(-L // ac_)
        assert info.gram_units == n_gram
        assert abs(info.ns_flops - sym) <= 1e-9 * sym
        assert info.gemm_tiles[0] == gram and info.gemm_tiles[1] == poly
        assert info.gemm_tiles[2] == apply
        assert info.workspace_bytes > 0
        # Launches per iteration: Gram, poly, apply for units as printed; with
        # Gram-space units also the Q / T and the A products (none in the
        # last iteration), and no Gram after the first iteration when every
        # unit is a Gram-space one.
        # K = 5: 3 K as printed; with both kinds of unit 5, 5, 4 (segment of
        # 3: no A update in its last iteration) then 5, 4; with Gram-space
        # units only 4, 3, 3, 4, 3 (a Gram only where a segment starts).
        if n_gram == 0:
            assert info.gemm_launches == 15
        else:
            assert info.gemm_launches == (17 if n_gram == len(units) else 23)
        # The apply reads Z row-major on every bf16 workload: per unit two Z
        # buffers (either layout) plus A and B, and Q[2] and T on a Gram-space
        # unit.
        if info.apply_nn:
            ws = 0
            for p, q in units:
                S, L = min(p, q), max(p, q)
                Sp, Lp = -(-S // 8) * 8, -(-L // 8) * 8
                g = S >= 128 and 4 * L >= 5 * S
                for n_el in (max(S * Lp, L * Sp),) * 2 + (S * Sp,) * (5 if g else 2):
                    ws = -(-(ws + n_el) // 128) * 128  # 256-byte aligned bf16 buffers
            assert info.workspace_bytes == 2 * ws


def test_describe_plan_qkv_numbers(lib):
    """2048 x 6144 with 8 column shards of 2048 x 768 (transposed: S = 768)."""
    mats = W.workload_matrices("qkv-2048x6144-bf16")
    blk = mb.describe_plan(mats, False)
    full = mb.describe_plan(mats, True)
    assert abs(blk.ns_dense_flops / 1e12 - 0.2295) < 5e-4
    assert abs(full.ns_dense_flops / 1e12 - 0.6013) < 5e-4
    # Every unit (the shards: S = 768, L = 2.7 S; the whole matrix: S = 2048,
    # L = 3 S) runs the Gram-space iteration in segments of 3 and 2:
    # 2 S(S+1)L + 14 S^2(S+1) + 4 S^2 L per unit; as printed, 5 (S(S+1)L +
    # S^2(S+1) + 2 S^2 L).
    assert full.gram_units == 1 and blk.gram_units == 8
    assert abs(blk.ns_flops / 1e12 - 0.1088) < 5e-4
    assert abs(full.ns_flops / 1e12 - 0.2750) < 5e-4
    opt = mb.options_default(gram_iteration=1)
    pb, pf = mb.describe_plan(mats, False, opt), mb.describe_plan(mats, True, opt)
    assert pb.gram_units == pf.gram_units == 0
    assert abs(pb.ns_flops / 1e12 - 0.1632) < 5e-4 and abs(pf.ns_flops / 1e12 - 0.4296) < 5e-4


@pytest.mark.parametrize("policy,shape,square", [
    (1, (128, 128), 128), (2, (256, 128), 128), (3, (256, 256), 256), (4, (128, 128), 128),
    (5, (256, 128), 128), (6, (256, 256), 256), (7, (128, 128), 128), (8, (128, 128), 128),
    (9, (256, 128), 128), (10, (256, 256), 256), (11, (192, 256), 192), (12, (256, 192), 192),
    (13, (192, 192), 192), (14, (256, 256), 256), (15, (192, 256), 192), (16, (256, 192), 192)])
def test_tile_policy_forces_shape(lib, policy, shape, square):
    """A forced tile shape reaches the apply product; the symmetric products
    take the nearest square shape."""
    mats = W.workload_matrices("qkv-2048x6144-bf16")
    info = mb.describe_plan(mats, False, mb.options_default(tile_policy=policy))
    assert (info.gemm_tile_rows[2], info.gemm_tile_cols[2]) == shape
    assert (info.gemm_tile_rows[0], info.gemm_tile_cols[0]) == (square, square)
    assert (info.gemm_tile_rows[1], info.gemm_tile_cols[1]) == (square, square)


def test_tile_model_choices(lib):
    """The planner's time model picks tiles that fill the 256 CUs: the
    2048 x 768 shards' apply takes 192 x 256 tiles (256 of them), the whole
    2048 x 6144 matrix's apply 256 x 192 tiles (256), and the large models
    256 x 256 tiles."""
    mats = W.workload_matrices("qkv-2048x6144-bf16")
    blk, full = mb.describe_plan(mats, False), mb.describe_plan(mats, True)
    assert (blk.gemm_tile_rows[2], blk.gemm_tile_cols[2], blk.gemm_tiles[2]) == (192, 256, 256)
    assert (full.gemm_tile_rows[2], full.gemm_tile_cols[2], full.gemm_tiles[2]) == (256, 192, 256)
    big = mb.describe_plan(W.workload_matrices("llama-32L-d4096-bf16"), False)
    assert list(big.gemm_tile_rows) == [256, 256, 256] and list(big.gemm_tile_cols) == [256, 256, 256]
    # fp32 NS operands: register K loop shapes only.
    f32 = mb.describe_plan(mats, False, mb.options_default(ns_dtype=mb.F32))
    assert f32.gemm_tile_rows[2] in (128, 256) and f32.gemm_tile_cols[2] in (128, 256)


def test_describe_plan_rejects_bad_grid(lib):
    with pytest.raises(mb.MuonBPError):
        mb.describe_plan([(10, 10, 3, 1)], False)


def test_three_launches_per_iteration(lib):
    """Three grouped launches per iteration as printed (gram_iteration = 1);
    the Gram-space schedule of the other modes is counted in
    test_describe_plan_counts_and_flops."""
    opt = mb.options_default(gram_iteration=1)
    for name in ("qkv-2048x6144-bf16", "llama-32L-d4096-bf16"):
        for full in (False, True):
            info = mb.describe_plan(W.workload_matrices(name), full, opt)
            assert info.gemm_launches == 3 * 5
    info = mb.describe_plan([(64, 64, 1, 1)], False, mb.options_default(ns_steps=0))
    assert info.gemm_launches == 0


def test_gram_iteration_modes(lib):
    """Which units run the Gram-space iteration: mode 0 from S >= 128 and
    L >= 1.25 S, mode 1 none, mode 2 every unit that allows it; never with
    K < 2, fp32 NS or the transposed-copy apply; an out-of-range mode is
    refused."""
    mats = [(1024, 1280, 1, 1), (1024, 1272, 1, 1), (1016, 4096, 1, 1), (4096, 1024, 1, 1), (296, 704, 1, 1),
            (120, 800, 1, 1)]
    gram = [0, 2, 3, 4]  # 1272 < 1.25 S; 120 < 128
    info = lambda **kw: mb.describe_plan(mats, True, mb.options_default(**kw))
    assert info().gram_units == len(gram)
    assert info(gram_iteration=1).gram_units == 0
    assert info(gram_iteration=2).gram_units == 6
    assert info(gram_iteration=2, ns_steps=1).gram_units == 0
    assert info(gram_iteration=2, ns_dtype=mb.F32).gram_units == 0
    assert info(gram_iteration=2, apply_mode=1).gram_units == 0
    # Three more S x Sp bf16 buffers (Q[2], T) per Gram-space unit, each
    # rounded up to 256 bytes.
    extra = sum(-(-min(mats[i][:2]) ** 2 // 128) * 128 for i in gram)
    assert info().workspace_bytes - info(gram_iteration=1).workspace_bytes == 2 * 3 * extra
    with pytest.raises(mb.MuonBPError):
        info(gram_iteration=3)


def test_in_place_units_skip_the_pack(lib):
    """Untransposed units whose NS input is the bf16 momentum itself are not
    packed (their first Gram and apply read the momentum in place); a
    transposed unit, a Nesterov blend, fp32 state or NS, K = 0, the
    transposed-copy apply or a column count off the 16-byte grid keeps the
    pack."""
    mats = [(512, 4096, 1, 1), (4096, 512, 1, 1), (1024, 1024, 1, 1), (1792, 4096, 8, 1), (4096, 1792, 1, 8)]
    elems = [r * c for r, c, _, _ in mats]
    packed_full = elems[1] + elems[4]  # the transposed ones
    info = lambda full=True, **kw: mb.describe_plan(mats, full, mb.options_default(**kw))
    assert info().pack_elements == packed_full
    # Block plan: the 8x1 grid's 224 x 4096 blocks are untransposed, the 1x8
    # grid's 4096 x 224 blocks transposed.
    assert info(False).pack_elements == packed_full
    for kw in (dict(nesterov=1), dict(state_dtype=mb.F32), dict(ns_dtype=mb.F32), dict(ns_steps=0),
               dict(apply_mode=1)):
        assert info(**kw).pack_elements == sum(elems), kw
    # In place from one iteration up, with or without the Gram-space iteration.
    assert info(ns_steps=1).pack_elements == packed_full
    assert info(gram_iteration=1).pack_elements == packed_full
    # Same launches and workspace: only the first products' operands move.
    assert info().gemm_launches == info(nesterov=1).gemm_launches
    assert info().workspace_bytes == info(nesterov=1).workspace_bytes
    # Rows of the momentum not on 16-byte boundaries (1004 columns).
    assert mb.describe_plan([(256, 1004, 1, 1)], True, mb.options_default()).pack_elements == 256 * 1004


def test_k_split_applies_to_dma_pipeline_only(lib):
    """A forced K split reaches the interleaved DMA kernels (bf16, K a
    multiple of 8); other kernels never split."""
    mats = W.workload_matrices("qkv-2048x6144-bf16")
    info = mb.describe_plan(mats, False, mb.options_default(tile_policy=8, k_split=4))
    assert list(info.gemm_split) == [4, 4, 4]
    info = mb.describe_plan(mats, False, mb.options_default(tile_policy=1, k_split=4))
    assert list(info.gemm_split) == [1, 1, 1]
    info = mb.describe_plan(mats, False, mb.options_default(ns_dtype=mb.F32, k_split=4))
    assert list(info.gemm_split) == [1, 1, 1]
    # k_split 1: never split.
    for name in W.WORKLOADS:
        for full in (False, True):
            info = mb.describe_plan(W.workload_matrices(name), full, mb.options_default(k_split=1))
            assert list(info.gemm_split) == [1, 1, 1]
    # The planner's choice (k_split 0) splits only launches that leave most
    # CUs idle with a long K loop: of the workloads, the whole 2048 x 6144
    # matrix's Gram (136 tiles, K = 6144); its A.A (K = 2048) stays whole.
    for name in W.WORKLOADS:
        for full in (False, True):
            info = mb.describe_plan(W.workload_matrices(name), full)
            want = [3, 1, 1] if (name == "qkv-2048x6144-bf16" and full) else [1, 1, 1]
            assert list(info.gemm_split) == want, (name, full)


def test_coefficient_table_plans_one_polynomial_per_entry(lib):
    """A per-iteration table changes only the polynomial descriptors: the
    same tiles, launches and flops as the constant quintic."""
    mats = W.workload_matrices("qkv-2048x6144-bf16")
    base = mb.describe_plan(mats, False)
    tab = mb.describe_plan(mats, False, mb.options_default(coeffs=[(3.0, -3.2, 1.2)] * 3))
    assert list(base.gemm_tiles) == list(tab.gemm_tiles)
    assert base.gemm_launches == tab.gemm_launches and base.ns_flops == tab.ns_flops


def test_apply_reads_z_row_major_where_the_dma_kernel_runs(lib):
    """bf16 NS with the interleaved DMA kernel on the apply: no Z^T operand;
    apply_mode 1, fp32 NS or a register-loop tile policy keep Z^T."""
    mats = [(2048, 6144, 1, 8)]
    for full in (0, 1):
        assert mb.describe_plan(mats, full, mb.options_default()).apply_nn == 1
        assert mb.describe_plan(mats, full, mb.options_default(apply_mode=1)).apply_nn == 0
        assert mb.describe_plan(mats, full, mb.options_default(ns_dtype=0)).apply_nn == 0
        assert mb.describe_plan(mats, full, mb.options_default(tile_policy=3)).apply_nn == 0
        # Policy 6 is an alias of 10 (interleaved DMA, 256 x 256 tiles).
        assert mb.describe_plan(mats, full, mb.options_default(tile_policy=6)).apply_nn == \
            mb.describe_plan(mats, full, mb.options_default(tile_policy=10)).apply_nn
        assert mb.describe_plan(mats, full, mb.options_default(tile_policy=11)).apply_nn == 1


def test_schedules_match_the_oracle(lib):
    from oracle import scalar_oracle as S
    T = 1000
    for t in list(range(0, 40)) + list(range(480, 520)) + list(range(780, 1010)):
        for warm in (0, 10):
            assert mb.lr_cosine(t, T, 3e-3, 3e-5, warm) == pytest.approx(
                S.lr_cosine(t, T, 3e-3, 3e-5, warm), rel=1e-14, abs=1e-18)
            for decay in (0, 200):
                assert mb.lr_wsd(t, T, 2e-2, 4.2e-5, warm, decay) == pytest.approx(
                    S.lr_wsd(t, T, 2e-2, 4.2e-5, warm, decay), rel=1e-14, abs=1e-18)


def test_adamw_options_default(lib):
    o = mb.adamw_options_default()
    assert (o.beta1, o.beta2) == pytest.approx((0.9, 0.95))
    assert o.eps == pytest.approx(1e-8) and o.weight_decay == pytest.approx(0.1)
    assert o.max_grad_norm == 1.0 and o.param_dtype == mb.BF16 and o.stream_hint == 0
    assert o.algorithm == 0


def test_adamw_create_rejects_bad_arguments_before_gpu(lib):
    def create(sizes, **kw):
        arr = (ctypes.c_int64 * max(1, len(sizes)))(*sizes)
        ctx = ctypes.c_void_p()
        o = mb.adamw_options_default(**kw)
        st = lib.muonbp_adamw_create(arr, len(sizes), ctypes.byref(o), None, ctypes.byref(ctx))
        return st, ctx

    assert create([])[0] == 1
    assert create([10, 0])[0] == 2
    assert create([10, -3])[0] == 2
    assert create([10], beta1=1.0)[0] == 1
    assert create([10], beta2=-0.1)[0] == 1
    assert create([10], eps=-1.0)[0] == 1
    assert create([10], max_grad_norm=-1.0)[0] == 1
    assert create([10], weight_decay=float("nan"))[0] == 1
    assert create([10], stream_hint=3)[0] == 1
    assert create([10], algorithm=2)[0] == 1
    assert create([10], algorithm=-1)[0] == 1
    assert create([10], param_dtype=7)[0] == 3
    assert lib.muonbp_adamw_create(None, 1, None, None, ctypes.byref(ctypes.c_void_p())) == 1
    assert lib.muonbp_adamw_step(None, None, None, 0, 0.1) == 1
    assert lib.muonbp_adamw_grad_norm(None, None) == 1
    assert lib.muonbp_adamw_synchronize(None) == 1
    lib.muonbp_adamw_destroy(None)


def test_static_step_refuses_on_the_host(lib):
    """muonbp_step_static checks its arguments and the scratch its plan needs
    before any HIP call (no GPU here): NULL arrays are E_INVALID, a step
    larger than the static scratch array is E_TOO_LARGE.  The pointers are
    never dereferenced on these paths."""
    fake = (ctypes.c_void_p * 1)(256)
    mats = mb._mats([(4096, 8192, 1, 1)])
    args = (0, 1, 0.01, 0.02, 0.9, 0.0, None, None)
    assert lib.muonbp_step_static(None, 1, fake, fake, ctypes.c_void_p(256), *args) == 1
    assert lib.muonbp_step_static(mats, 1, None, fake, ctypes.c_void_p(256), *args) == 1
    assert lib.muonbp_step_static(mats, 1, fake, fake, None, *args) == 1
    assert lib.muonbp_step_static(mats, 1, fake, fake, ctypes.c_void_p(256), -1, 1, 0.01, 0.02,
                                  0.9, 0.0, None, None) == 1
    assert lib.muonbp_step_static(mats, 1, fake, fake, ctypes.c_void_p(256), *args) == 8
    assert mb.describe_plan([(4096, 8192, 1, 1)], True).static_scratch_bytes > mb.STATIC_SCRATCH_BYTES
    bad = (ctypes.c_void_p * 1)(257)  # not element-aligned
    assert lib.muonbp_step_static(mats, 1, bad, fake, ctypes.c_void_p(256), *args) == 1


def test_static_scratch_fits_the_qkv_workload(lib):
    """The static scratch array is sized for one 2048 x 6144 matrix in
    2048 x 768 shards, in both plans."""
    mats = W.workload_matrices("qkv-2048x6144-bf16")
    for full in (False, True):
        info = mb.describe_plan(mats, full)
        assert info.workspace_bytes < info.static_scratch_bytes <= mb.STATIC_SCRATCH_BYTES

