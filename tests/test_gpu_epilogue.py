"""GPU: the fused epilogue (bias + ReLU, 2x2 max-pool) of every variant and
split count gives exactly the unfused sequence -- the same plan's convolution,
then ReLU, then the pool, applied to its fp32 output -- on OIHW and on
prepacked weights, and, anchored to the oracle, max-pool(ReLU(exact conv))
within the tolerance."""
import numpy as np
import pytest

import oracle
import workloads
from gpu_common import dev, note, random_case, torch_cuda

pytestmark = pytest.mark.gpu

EPIS = (1, 2, 3)  # RELU, MAXPOOL2, both


@pytest.fixture(scope="module")
def ilpm():
    torch_cuda()
    import paper_1909_02765_amd as m
    oracle.set_threads(16)
    return m


def pool_relu_np(y, epi):
    """ReLU and/or 2x2 max-pool (floor) of a [1,C,H,W] float32 array, exactly."""
    if epi & 1:
        y = np.maximum(y, np.float32(0))
    if epi & 2:
        _, c, h, w = y.shape
        y = y[:, :, : h // 2 * 2, : w // 2 * 2].reshape(1, c, h // 2, 2, w // 2, 2).max(axis=(3, 5))
    return y


def all_plans(ilpm, c_in, h, w, c_out, k, s, p):
    plans = []
    for v in range(ilpm.num_variants(ilpm.PATH_DIRECT)):
        try:
            plans.append(ilpm.plan_variant(c_in, h, w, c_out, k, s, p, ilpm.PATH_DIRECT, v))
        except ilpm.IlpmError:
            pass
    for v in range(ilpm.num_variants(ilpm.PATH_IGEMM)):
        seen = set()
        for splits in (1, 0, 3):
            try:
                q = ilpm.plan_variant(c_in, h, w, c_out, k, s, p, ilpm.PATH_IGEMM, v, splits)
            except ilpm.IlpmError:
                continue
            if q.splits not in seen:
                seen.add(q.splits)
                plans.append(q)
    return plans


def check_case(ilpm, name, x, w, b, s, p, skip_slow=False):
    torch = torch_cuda()
    c_out, c_in, k, _ = w.shape
    h, wd = x.shape[2], x.shape[3]
    xd, wdv, bd = dev(x), dev(w), dev(b)
    for plan in all_plans(ilpm, c_in, h, wd, c_out, k, s, p):
        if skip_slow and plan.path == ilpm.PATH_DIRECT and plan.variant == 1:
            continue
        unfused = ilpm.conv2d(xd, wdv, bd, s, p, plan=plan)
        packed = ilpm.prepack_weights(wdv, plan)
        torch.cuda.synchronize()
        base = unfused.cpu().numpy()
        for epi in EPIS:
            note(f"[epilogue] {name} path={plan.path} v={plan.variant} splits={plan.splits} epi={epi}")
            got = ilpm.conv2d_epilogue(xd, wdv, bd, s, p, epi, plan=plan)
            torch.cuda.synchronize()
            label = f"{name} plan {plan.path}/{plan.variant}/{plan.splits} epi {epi}"
            np.testing.assert_array_equal(got.cpu().numpy(), pool_relu_np(base, epi), err_msg=label)
            note(f"[epilogue prepacked] {name} path={plan.path} v={plan.variant} splits={plan.splits} epi={epi}")
            got = ilpm.conv2d_prepacked_epilogue(xd, packed, c_out, k, bd, s, p, epi, plan=plan)
            torch.cuda.synchronize()
            np.testing.assert_array_equal(got.cpu().numpy(), pool_relu_np(base, epi), err_msg=label + " prepacked")


@pytest.mark.parametrize("case", workloads.ALL_CASES, ids=lambda c: c.name)
def test_epilogue_matches_unfused(ilpm, case):
    x, w, b = case.inputs()
    big = case.c_in * case.c_out * case.h * case.w > 5e7
    check_case(ilpm, case.name, x, w, b, case.stride, case.pad, skip_slow=big)


def test_epilogue_ragged(ilpm):
    """Odd output sizes (the pool drops the last row/column), partial tiles,
    and channel counts that fill no tile exactly."""
    for seed, (c_in, h, w_, c_out, k, s, p) in enumerate([(13, 17, 19, 40, 3, 1, 1), (37, 9, 9, 70, 1, 1, 0),
                                                         (21, 11, 10, 33, 5, 1, 2), (29, 15, 15, 17, 3, 2, 1)]):
        x, w, b = random_case(8000 + 10 * seed, c_in, h, w_, c_out, k)
        check_case(ilpm, f"ragged{seed}", x, w, b, s, p)


def test_epilogue_against_oracle(ilpm):
    """Default plan, both bits: max-pool(ReLU(exact conv)) within the
    tolerance of the window element the maximum comes from (max and ReLU are
    1-Lipschitz, so the largest window tolerance bounds the difference)."""
    torch = torch_cuda()
    for case in (workloads.VGG_EARLY, workloads.RESNET_CONV2, workloads.RESNET_CONV5):
        x, w, b = case.inputs()
        ref, sab = oracle.conv2d_f64(x, w, b, case.stride, case.pad)
        tol = oracle.tolerance(sab, case.c_in, case.k)
        want = pool_relu_np(ref, 3)
        tw = pool_relu_np(tol, 2)  # largest tolerance per window
        note(f"[epilogue-oracle] {case.name}")
        got = ilpm.conv2d_epilogue(dev(x), dev(w), dev(b), case.stride, case.pad, 3)
        torch.cuda.synchronize()
        err = np.abs(got.cpu().numpy().astype(np.float64) - want)
        assert (err <= tw).all(), f"{case.name}: worst {np.max(err / tw)}"


def test_pooled_tile_writes_only_the_pooled_output(ilpm):
    """One-split plans whose tiles have even sides pool inside the kernel: NaN
    canaries around the pooled output survive, the values equal conv -> ReLU
    -> pool of the same plan, and for the 14x14-tile variants (which pool in
    the workgroup) a NaN-filled registered workspace is left untouched."""
    torch = torch_cuda()
    guard = 4096
    in_kernel = {"k3s1_t14x14_co64_cc16_pf", "k3s1_t14x14_co32_k2", "k3s1_t14x14_co64",
                 "k3s1_t14x14_co64_cc16_pf_sc1", "k3s1_t14x14_co64_cc4_sc1", "k3s1_t14x14_co32_k2_sc1"}
    ws = torch.full((1 << 22,), float("nan"), device="cuda", dtype=torch.float32)
    ilpm.set_workspace(ws)
    try:
        for seed, (c_in, h, w_, c_out) in enumerate([(64, 30, 30, 70), (32, 17, 19, 40), (48, 28, 29, 64)]):
            x, w, b = random_case(8600 + 10 * seed, c_in, h, w_, c_out, 3)
            xd, wdv, bd = dev(x), dev(w), dev(b)
            ho, wo = h // 2, w_ // 2
            n = c_out * ho * wo
            for v in range(ilpm.num_variants(ilpm.PATH_IGEMM)):
                info = ilpm.variant_info(ilpm.PATH_IGEMM, v)
                if info["k"] != 3 or info["stride"] != 1 or info["tile_h"] % 2 or info["tile_w"] % 2:
                    continue
                try:
                    plan = ilpm.plan_variant(c_in, h, w_, c_out, 3, 1, 1, ilpm.PATH_IGEMM, v, 1)
                except ilpm.IlpmError:
                    continue
                name = ilpm.variant_name(ilpm.PATH_IGEMM, v)
                note(f"[pooled tile] shape {(c_in, h, w_, c_out)} v={v} {name}")
                base = ilpm.conv2d(xd, wdv, bd, 1, 1, plan=plan)
                torch.cuda.synchronize()
                want = pool_relu_np(base.cpu().numpy(), 3)
                ws.fill_(float("nan"))
                buf = torch.full((n + 2 * guard,), float("nan"), device="cuda", dtype=torch.float32)
                out = buf[guard:guard + n].view(1, c_out, ho, wo)
                ilpm.conv2d_epilogue(xd, wdv, bd, 1, 1, ilpm.EPI_RELU | ilpm.EPI_MAXPOOL2, plan=plan, out=out)
                torch.cuda.synchronize()
                assert torch.isnan(buf[:guard]).all() and torch.isnan(buf[guard + n:]).all(), name
                np.testing.assert_array_equal(out.cpu().numpy(), want, err_msg=name)
                if name in in_kernel:
                    assert torch.isnan(ws).all(), f"{name}: the pooled tile went through the workspace"
                # the same with prepacked weights (the kernel pools in the workgroup too)
                packed = ilpm.prepack_weights(wdv, plan)
                buf.fill_(float("nan"))
                note(f"[pooled tile prepacked] shape {(c_in, h, w_, c_out)} v={v} {name}")
                ilpm.conv2d_prepacked_epilogue(xd, packed, c_out, 3, bd, 1, 1, ilpm.EPI_RELU | ilpm.EPI_MAXPOOL2,
                                               plan=plan, out=out)
                torch.cuda.synchronize()
                assert torch.isnan(buf[:guard]).all() and torch.isnan(buf[guard + n:]).all(), name + " prepacked"
                np.testing.assert_array_equal(out.cpu().numpy(), want, err_msg=name + " prepacked")
                if name in in_kernel:
                    assert torch.isnan(ws).all(), f"{name} prepacked: the pooled tile went through the workspace"
    finally:
        torch.cuda.synchronize()
        ilpm.set_workspace(None)


def test_device_scope_store_variants_match_their_plain_twins(ilpm):
    """The `_sc1` variants differ from their plain twins only in the cache
    policy of the output stores: same bits, plain and with ReLU + 2x2
    max-pool (in the workgroup or after split partial sums), on OIHW and on
    prepacked weights, on shapes that leave partial tiles."""
    torch = torch_cuda()
    names = {ilpm.variant_name(ilpm.PATH_IGEMM, v): v for v in range(ilpm.num_variants(ilpm.PATH_IGEMM))}
    pairs = [(names[n[:-4]], v) for n, v in names.items() if n.endswith("_sc1") and n[:-4] in names]
    assert len(pairs) >= 5
    for seed, (c_in, h, w_, c_out) in enumerate([(64, 30, 30, 70), (48, 17, 23, 40)]):
        x, w, b = random_case(8800 + 10 * seed, c_in, h, w_, c_out, 3)
        xd, wdv, bd = dev(x), dev(w), dev(b)
        for v_plain, v_sc1 in pairs:
            for splits in (1, 3):
                try:
                    p_plain = ilpm.plan_variant(c_in, h, w_, c_out, 3, 1, 1, ilpm.PATH_IGEMM, v_plain, splits)
                    p_sc1 = ilpm.plan_variant(c_in, h, w_, c_out, 3, 1, 1, ilpm.PATH_IGEMM, v_sc1, splits)
                except ilpm.IlpmError:
                    continue
                label = f"{ilpm.variant_name(ilpm.PATH_IGEMM, v_sc1)} x{p_sc1.splits} {(c_in, h, w_, c_out)}"
                note(f"[sc1 twin] {label}")
                for epi in (0, 3):
                    want = ilpm.conv2d_epilogue(xd, wdv, bd, 1, 1, epi, plan=p_plain)
                    got = ilpm.conv2d_epilogue(xd, wdv, bd, 1, 1, epi, plan=p_sc1)
                    packed = ilpm.prepack_weights(wdv, p_sc1)
                    got_pk = ilpm.conv2d_prepacked_epilogue(xd, packed, c_out, 3, bd, 1, 1, epi, plan=p_sc1)
                    torch.cuda.synchronize()
                    np.testing.assert_array_equal(got.cpu().numpy(), want.cpu().numpy(), err_msg=f"{label} epi {epi}")
                    np.testing.assert_array_equal(got_pk.cpu().numpy(), want.cpu().numpy(),
                                                  err_msg=f"{label} epi {epi} prepacked")
