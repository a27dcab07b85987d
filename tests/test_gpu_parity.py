"""GPU parity: the HIP path (through the C ABI) against the CPU oracle, element
by element, within 1e-4 * (1 + S / (C_in*K*K)); bit for bit where every
partial sum is exactly representable (small-integer tensors)."""
import numpy as np
import pytest

import oracle
import workloads
from gpu_common import (assert_matches, dev, note, random_case, run_conv, small_int_case, torch_cuda)

pytestmark = pytest.mark.gpu

CASES = workloads.ALL_CASES
_ORACLE = {}


@pytest.fixture(scope="module")
def ilpm():
    torch_cuda()
    import paper_1909_02765_amd as m
    oracle.set_threads(16)
    return m


def case_data(case):
    if case.name not in _ORACLE:
        x, w, b = case.inputs()
        ref, sab = oracle.conv2d_f64(x, w, b, case.stride, case.pad)
        _ORACLE[case.name] = (x, w, b, ref, sab)
    return _ORACLE[case.name]


def plans_for(ilpm, c_in, h, w, c_out, k, s, p):
    """Every compiled variant that accepts this shape, with one and several splits."""
    plans = []
    for v in range(ilpm.num_variants(ilpm.PATH_DIRECT)):
        try:
            plans.append(ilpm.plan_variant(c_in, h, w, c_out, k, s, p, ilpm.PATH_DIRECT, v))
        except ilpm.IlpmError:
            pass
    for v in range(ilpm.num_variants(ilpm.PATH_IGEMM)):
        info = ilpm.variant_info(ilpm.PATH_IGEMM, v)
        if info["k"] != k or info["stride"] != s:
            continue
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


def describe(plan):
    return (f"path={plan.path} v={plan.variant} tile={plan.tile_h}x{plan.tile_w} co={plan.co_tile} "
            f"splits={plan.splits} grid={plan.grid}")


@pytest.mark.parametrize("case", CASES, ids=lambda c: c.name)
def test_default_plan_full_output(ilpm, case):
    x, w, b, ref, sab = case_data(case)
    plan = ilpm.plan(case.c_in, case.h, case.w, case.c_out, case.k, case.stride, case.pad)
    note(f"[default] {case.name} {describe(plan)}")
    got = run_conv(x, w, b, case.stride, case.pad)
    assert_matches(got, ref, sab, case.c_in, case.k, case.name)


@pytest.mark.parametrize("case", CASES, ids=lambda c: c.name)
def test_every_variant_full_output(ilpm, case):
    x, w, b, ref, sab = case_data(case)
    plans = plans_for(ilpm, case.c_in, case.h, case.w, case.c_out, case.k, case.stride, case.pad)
    assert plans
    for plan in plans:
        if plan.path == ilpm.PATH_DIRECT and plan.variant == 1 and case.c_in * case.c_out * case.h * case.w > 50e6:
            continue  # the plain fallback kernel is covered on the smaller layers
        note(f"[variant] {case.name} {describe(plan)}")
        got = run_conv(x, w, b, case.stride, case.pad, plan=plan)
        assert_matches(got, ref, sab, case.c_in, case.k, f"{case.name} {describe(plan)}")


@pytest.mark.parametrize("case", CASES, ids=lambda c: c.name)
def test_small_integers_bit_exact(ilpm, case):
    """Integer tensors in [-2, 2]: every partial sum is an integer below 2^24, so
    any summation order gives the oracle's value exactly."""
    x, w, b = small_int_case(7000 + case.x_seed, case.c_in, case.h, case.w, case.c_out, case.k)
    ref, _ = oracle.conv2d_f64(x, w, b, case.stride, case.pad)
    assert np.abs(ref).max() < 2 ** 24
    for plan in [None] + plans_for(ilpm, case.c_in, case.h, case.w, case.c_out, case.k, case.stride, case.pad):
        if plan is not None and plan.path == ilpm.PATH_DIRECT and plan.variant == 1 and \
                case.c_in * case.c_out * case.h * case.w > 50e6:
            continue
        note(f"[exact] {case.name} {describe(plan) if plan is not None else 'default'}")
        got = run_conv(x, w, b, case.stride, case.pad, plan=plan)
        np.testing.assert_array_equal(got.astype(np.float64), ref)


def test_fuzz_small_shapes(ilpm):
    """Random small shapes: every variant that accepts each shape."""
    shapes = workloads.fuzz_shapes(2024, 40)
    for i, s in enumerate(shapes):
        x, w, b = random_case(100 + 3 * i, s["c_in"], s["h"], s["w"], s["c_out"], s["k"], bias=(i % 2 == 0))
        ref, sab = oracle.conv2d_f64(x, w, b, s["stride"], s["pad"])
        for plan in [None] + plans_for(ilpm, s["c_in"], s["h"], s["w"], s["c_out"], s["k"], s["stride"], s["pad"]):
            note(f"[fuzz {i}] {s} {describe(plan) if plan is not None else 'default'}")
            got = run_conv(x, w, b, s["stride"], s["pad"], plan=plan)
            assert_matches(got, ref, sab, s["c_in"], s["k"], f"fuzz {i} {s}")


def test_fuzz_matrix_core_ragged(ilpm):
    """Shapes that leave partial output tiles, partial channel stages and
    partial output-channel tiles for every matrix-core variant."""
    rng = np.random.default_rng(31)
    n = ilpm.num_variants(ilpm.PATH_IGEMM)
    for v in range(n):
        info = ilpm.variant_info(ilpm.PATH_IGEMM, v)
        k, s = info["k"], info["stride"]
        for j in range(4):
            c_in = int(rng.integers(1, 41))
            c_out = int(rng.integers(1, 150))
            h = int(rng.integers(1, 40))
            w = int(rng.integers(1, 40))
            p = int(rng.integers(0, k))
            if h + 2 * p < k or w + 2 * p < k:
                p = k
            x, wt, b = random_case(5000 + 10 * v + j, c_in, h, w, c_out, k, bias=(j % 2 == 1))
            ref, sab = oracle.conv2d_f64(x, wt, b, s, p)
            for splits in (1, 0, 2):
                try:
                    plan = ilpm.plan_variant(c_in, h, w, c_out, k, s, p, ilpm.PATH_IGEMM, v, splits)
                except ilpm.IlpmError:
                    continue
                note(f"[ragged] v={v} c_in={c_in} h={h} w={w} c_out={c_out} k={k} s={s} p={p} {describe(plan)}")
                got = run_conv(x, wt, b, s, p, plan=plan)
                assert_matches(got, ref, sab, c_in, k, f"ragged v={v} {describe(plan)}")


def split_variant(ilpm):
    """A 3x3 stride-1 matrix-core variant that takes any split count."""
    for v in range(ilpm.num_variants(ilpm.PATH_IGEMM)):
        if ilpm.variant_name(ilpm.PATH_IGEMM, v) == "k3s1_t7x7_co64_cc4":
            return v
    raise AssertionError("variant k3s1_t7x7_co64_cc4 missing")


def test_split_reduction_repeats_bitwise(ilpm):
    """A split plan run several times gives identical bits (the partial sums
    are added in a fixed order)."""
    case = workloads.RESNET_CONV4
    x, w, b, ref, sab = case_data(case)
    plan = ilpm.plan_variant(case.c_in, case.h, case.w, case.c_out, case.k, case.stride, case.pad,
                             ilpm.PATH_IGEMM, split_variant(ilpm), 8)
    assert plan.splits > 1
    note(f"[repeat] {describe(plan)}")
    outs = [run_conv(x, w, b, case.stride, case.pad, plan=plan) for _ in range(3)]
    for o in outs[1:]:
        np.testing.assert_array_equal(o, outs[0])
    assert_matches(outs[0], ref, sab, case.c_in, case.k, "repeat")


def test_registered_workspace(ilpm):
    torch = torch_cuda()
    case = workloads.RESNET_CONV4
    x, w, b, ref, sab = case_data(case)
    plan = ilpm.plan_variant(case.c_in, case.h, case.w, case.c_out, case.k, case.stride, case.pad,
                             ilpm.PATH_IGEMM, split_variant(ilpm), 4)
    assert plan.workspace_bytes > 0
    small = torch.empty(1024, dtype=torch.float32, device="cuda")
    big = torch.empty((plan.workspace_bytes + 3) // 4 + 64, dtype=torch.float32, device="cuda")
    try:
        ilpm.set_workspace(small)
        with pytest.raises(ilpm.IlpmError) as e:
            run_conv(x, w, b, case.stride, case.pad, plan=plan)
        assert e.value.status == ilpm.ERR_WORKSPACE
        ilpm.set_workspace(big)
        note("[workspace] registered")
        got = run_conv(x, w, b, case.stride, case.pad, plan=plan)
        assert_matches(got, ref, sab, case.c_in, case.k, "registered workspace")
    finally:
        ilpm.set_workspace(None)
        torch.cuda.synchronize()


def test_non_default_stream(ilpm):
    torch = torch_cuda()
    case = workloads.RESNET_STRIDED
    x, w, b, ref, sab = case_data(case)
    s = torch.cuda.Stream()
    note("[stream] side stream")
    with torch.cuda.stream(s):
        got = run_conv(x, w, b, case.stride, case.pad, stream=s)
    assert_matches(got, ref, sab, case.c_in, case.k, "side stream")


def test_bad_arguments_raise(ilpm):
    torch = torch_cuda()
    x = torch.zeros((1, 4, 8, 8), device="cuda")
    w = torch.zeros((4, 4, 3, 3), device="cuda")
    # an output aliasing the input is refused before anything is launched
    rc = ilpm.lib.ilpm_conv2d_fwd(x.data_ptr(), w.data_ptr(), None, 4, 8, 8, 4, 3, 1, 1, x.data_ptr(), None)
    assert rc == ilpm.ERR_INVALID_ARG
    with pytest.raises(TypeError):
        ilpm.conv2d(x.double(), w, None)


@pytest.mark.parametrize("case", [workloads.RESNET_CONV4, workloads.TINY], ids=lambda c: c.name)
def test_graph_replay_matches_eager(ilpm, case):
    """Calls captured in a HIP graph and replayed several times, with eager work
    and a synchronisation between replays, reproduce the eager result bit for
    bit (one plan with the split-sum kernel, one without)."""
    torch = torch_cuda()
    x, w, b, ref, sab = case_data(case)
    xd, wd, bd = dev(x), dev(w), dev(b)
    ho = ilpm.out_size(case.h, case.k, case.stride, case.pad)
    wo = ilpm.out_size(case.w, case.k, case.stride, case.pad)
    out = torch.empty((1, case.c_out, ho, wo), device="cuda", dtype=torch.float32)
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    note(f"[graph] {case.name} capture")
    with torch.cuda.stream(s):
        launch = ilpm.conv2d_launcher(xd, wd, bd, case.stride, case.pad, out)
        launch()
        torch.cuda.synchronize()
        eager = out.cpu().numpy().copy()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=s):
            launch()
    torch.cuda.synchronize()
    assert_matches(eager, ref, sab, case.c_in, case.k, "eager before capture")
    for i in range(4):
        note(f"[graph] {case.name} replay {i}")
        out.fill_(float("nan"))
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        np.testing.assert_array_equal(out.cpu().numpy(), eager)


def _prepacked_vs_oihw(ilpm, x, w, b, stride, pad, plan, label):
    torch = torch_cuda()
    c_out, c_in, k, _ = w.shape
    xd, wd, bd = dev(x), dev(w), dev(b)
    ho, wo = ilpm.out_size(x.shape[2], k, stride, pad), ilpm.out_size(x.shape[3], k, stride, pad)
    note(f"[prepacked] {label} {describe(plan)}")
    want = ilpm.conv2d(xd, wd, bd, stride, pad, plan=plan)
    packed = ilpm.prepack_weights(wd, plan)
    assert packed.numel() * 4 == ilpm.prepacked_size(plan, c_in, c_out, k)
    got = ilpm.conv2d_prepacked(xd, packed, c_out, k, bd, stride, pad, plan=plan)
    torch.cuda.synchronize()
    np.testing.assert_array_equal(got.cpu().numpy(), want.cpu().numpy(), err_msg=f"{label} {describe(plan)}")
    assert got.shape == (1, c_out, ho, wo)


@pytest.mark.parametrize("case", CASES, ids=lambda c: c.name)
def test_prepacked_matches_oihw_bitwise(ilpm, case):
    """Every variant run on prepacked weights gives exactly the bits of the same
    plan on the OIHW weights (the packing moves data, it changes no
    arithmetic); the OIHW path is checked against the oracle elsewhere."""
    x, w, b, ref, sab = case_data(case)
    for plan in plans_for(ilpm, case.c_in, case.h, case.w, case.c_out, case.k, case.stride, case.pad):
        if plan.path == ilpm.PATH_DIRECT and plan.variant == 1 and case.c_in * case.c_out * case.h * case.w > 5e7:
            continue  # the plain-global direct kernel is slow on the large layers; it reads OIHW either way
        _prepacked_vs_oihw(ilpm, x, w, b, case.stride, case.pad, plan, case.name)


def test_prepacked_ragged_channels(ilpm):
    """Channel counts that leave partial output-channel tiles and partial
    input-channel chunks (the packed layout's zero padding), against the
    oracle as well."""
    for seed, (c_in, h, w_, c_out, k, s, p) in enumerate([(13, 17, 19, 40, 3, 1, 1), (37, 9, 9, 70, 1, 1, 0),
                                                         (21, 11, 10, 33, 5, 1, 2), (29, 15, 15, 17, 3, 2, 1)]):
        x, w, b = random_case(7000 + 10 * seed, c_in, h, w_, c_out, k)
        ref, sab = oracle.conv2d_f64(x, w, b, s, p)
        for v in range(ilpm.num_variants(ilpm.PATH_IGEMM)):
            info = ilpm.variant_info(ilpm.PATH_IGEMM, v)
            if info["k"] != k or info["stride"] != s:
                continue
            for splits in (1, 0):
                try:
                    plan = ilpm.plan_variant(c_in, h, w_, c_out, k, s, p, ilpm.PATH_IGEMM, v, splits)
                except ilpm.IlpmError:
                    continue
                _prepacked_vs_oihw(ilpm, x, w, b, s, p, plan, f"ragged{seed}")
                torch = torch_cuda()
                packed = ilpm.prepack_weights(dev(w), plan)
                got = ilpm.conv2d_prepacked(dev(x), packed, c_out, k, dev(b), s, p, plan=plan)
                torch.cuda.synchronize()
                assert_matches(got.cpu().numpy(), ref, sab, c_in, k, f"prepacked ragged{seed} v{v}")


def test_one_by_one_consecutive_channels(ilpm):
    """1x1 variants, including those whose lanes take consecutive input
    channels (one 16-byte weight load per four channels; planned only for
    C_in a multiple of 4): partial channel stages, partial output-channel
    tiles and ragged planes, split and not, on OIHW and prepacked weights
    (the same bits) and against the oracle."""
    torch = torch_cuda()
    ones = [v for v in range(ilpm.num_variants(ilpm.PATH_IGEMM)) if ilpm.variant_info(ilpm.PATH_IGEMM, v)["k"] == 1]
    assert ones
    ran = set()
    for seed, (c_in, h, w_, c_out) in enumerate([(4, 5, 9, 20), (12, 7, 7, 33), (36, 9, 11, 70), (68, 4, 6, 17),
                                                 (132, 7, 7, 48)]):
        x, w, b = random_case(7500 + 10 * seed, c_in, h, w_, c_out, 1, bias=(seed % 2 == 0))
        ref, sab = oracle.conv2d_f64(x, w, b, 1, 0)
        for v in ones:
            for splits in (1, 0, 2):
                try:
                    plan = ilpm.plan_variant(c_in, h, w_, c_out, 1, 1, 0, ilpm.PATH_IGEMM, v, splits)
                except ilpm.IlpmError:
                    continue
                note(f"[1x1] {(c_in, h, w_, c_out)} {describe(plan)}")
                got = run_conv(x, w, b, 1, 0, plan=plan)
                assert_matches(got, ref, sab, c_in, 1, f"1x1 {(c_in, h, w_, c_out)} {describe(plan)}")
                _prepacked_vs_oihw(ilpm, x, w, b, 1, 0, plan, f"1x1 {(c_in, h, w_, c_out)}")
                ran.add(v)
    assert ran == set(ones)


def test_wide_channels_many_splits(ilpm):
    """Channel counts that are not multiples of the stage size, split into
    uneven ranges across many workgroups (the small-layer plans).  The values
    follow the workloads' recipe (inputs uniform[0,1], He-normal weights):
    with thousands of terms per output, weights of unit scale would make the
    outputs large and the plain fp32 rounding of a long sum alone exceed the
    tolerance, which is stated for that recipe."""
    for j, (c_in, h, w_, c_out, k, s, p) in enumerate([(300, 9, 9, 200, 3, 1, 1), (513, 7, 7, 130, 1, 1, 0),
                                                       (257, 12, 12, 96, 5, 1, 2), (190, 15, 13, 70, 3, 2, 1)]):
        x = workloads.uniform(6100 + 10 * j, (1, c_in, h, w_), 0.0, 1.0)
        w = workloads.normal(6101 + 10 * j, (c_out, c_in, k, k), 0.0, workloads.he_std(c_in, k))
        b = workloads.normal(6102 + 10 * j, (c_out,), 0.0, 0.01) if j % 2 == 0 else None
        ref, sab = oracle.conv2d_f64(x, w, b, s, p)
        for v in range(ilpm.num_variants(ilpm.PATH_IGEMM)):
            info = ilpm.variant_info(ilpm.PATH_IGEMM, v)
            if info["k"] != k or info["stride"] != s:
                continue
            seen = set()
            for splits in (1, 5, 7, 0, 64):
                try:
                    plan = ilpm.plan_variant(c_in, h, w_, c_out, k, s, p, ilpm.PATH_IGEMM, v, splits)
                except ilpm.IlpmError:
                    continue
                if plan.splits in seen:
                    continue
                seen.add(plan.splits)
                note(f"[wide {j}] v={v} {describe(plan)}")
                got = run_conv(x, w, b, s, p, plan=plan)
                assert_matches(got, ref, sab, c_in, k, f"wide {j} v={v} {describe(plan)}")


def test_fixed_stage_variants_ragged(ilpm):
    """The three-buffer variants (built for an exact stage count, loads of the
    stage after next in flight): one and two splits, the last channel chunk
    partly filled, partial output-channel and spatial tiles, with and without
    bias; against the oracle, and prepacked weights against OIHW bit for bit."""
    rng = np.random.default_rng(41)
    for v in range(ilpm.num_variants(ilpm.PATH_IGEMM)):
        info = ilpm.variant_info(ilpm.PATH_IGEMM, v)
        if not info["stages"]:
            continue
        k, s, ns, cc = info["k"], info["stride"], info["stages"], info["ci_chunk"]
        for j, splits in enumerate((1, 2)):
            c_in = ns * cc * splits - int(rng.integers(0, cc))
            c_out = int(rng.integers(17, 90))
            h = int(rng.integers(5, 19))
            w_ = int(rng.integers(5, 19))
            p = k // 2
            x = workloads.uniform(8100 + 10 * v + j, (1, c_in, h, w_), 0.0, 1.0)
            wt = workloads.normal(8101 + 10 * v + j, (c_out, c_in, k, k), 0.0, workloads.he_std(c_in, k))
            b = workloads.normal(8102 + 10 * v + j, (c_out,), 0.0, 0.01) if j == 0 else None
            ref, sab = oracle.conv2d_f64(x, wt, b, s, p)
            plan = ilpm.plan_variant(c_in, h, w_, c_out, k, s, p, ilpm.PATH_IGEMM, v)
            assert plan.splits == splits
            note(f"[fixed-stage] v={v} c_in={c_in} h={h} w={w_} c_out={c_out} {describe(plan)}")
            got = run_conv(x, wt, b, s, p, plan=plan)
            assert_matches(got, ref, sab, c_in, k, f"fixed-stage v={v} {describe(plan)}")
            _prepacked_vs_oihw(ilpm, x, wt, b, s, p, plan, f"fixed-stage v={v}")


def test_progressive_first_stage_ragged(ilpm):
    """Variants whose first stage starts computing on its first four channels
    while the rest land (its halo in buffers of its own, waits counted per
    channel group): two to five stages, the last channel chunk partly filled,
    one and two splits, partial spatial and output-channel tiles, with and
    without bias; against the oracle, and prepacked weights against OIHW bit
    for bit (the prepacked kernel takes the same summation order)."""
    rng = np.random.default_rng(43)
    for v in range(ilpm.num_variants(ilpm.PATH_IGEMM)):
        info = ilpm.variant_info(ilpm.PATH_IGEMM, v)
        if not info["progressive_first"]:
            continue
        k, s, cc = info["k"], info["stride"], info["ci_chunk"]
        for j, (stages, splits) in enumerate(((2, 1), (5, 1), (4, 2))):
            c_in = stages * cc - int(rng.integers(0, cc - 1))
            c_out = int(rng.integers(17, 140))
            h = int(rng.integers(9, 45))
            w_ = int(rng.integers(9, 45))
            p = k // 2
            x = workloads.uniform(8300 + 10 * v + j, (1, c_in, h, w_), 0.0, 1.0)
            wt = workloads.normal(8301 + 10 * v + j, (c_out, c_in, k, k), 0.0, workloads.he_std(c_in, k))
            b = workloads.normal(8302 + 10 * v + j, (c_out,), 0.0, 0.01) if j != 1 else None
            ref, sab = oracle.conv2d_f64(x, wt, b, s, p)
            plan = ilpm.plan_variant(c_in, h, w_, c_out, k, s, p, ilpm.PATH_IGEMM, v, splits)
            assert plan.splits == splits
            note(f"[progressive] v={v} c_in={c_in} h={h} w={w_} c_out={c_out} {describe(plan)}")
            got = run_conv(x, wt, b, s, p, plan=plan)
            assert_matches(got, ref, sab, c_in, k, f"progressive v={v} {describe(plan)}")
            _prepacked_vs_oihw(ilpm, x, wt, b, s, p, plan, f"progressive v={v}")


def test_fused_split_sum_matches_kernel_bitwise(ilpm):
    """The fused split sum (the last workgroup of each tile adds the slices) and
    the separate split-sum kernel add the same slices in the same order, so
    every split plan gives the same bits either way.  Shapes alternate between
    calls, so a tile's arrival count left non-zero by one call would corrupt the
    next; each fused output is also checked against the oracle, and the ReLU
    epilogue takes the same path."""
    torch = torch_cuda()
    shapes = [(300, 9, 9, 200, 3, 1, 1), (96, 7, 7, 40, 1, 1, 0), (130, 11, 10, 70, 5, 1, 2),
              (70, 15, 13, 90, 3, 2, 1)]
    data = []
    for j, (c_in, h, w_, c_out, k, s, p) in enumerate(shapes):
        x = workloads.uniform(7100 + 10 * j, (1, c_in, h, w_), 0.0, 1.0)
        w = workloads.normal(7101 + 10 * j, (c_out, c_in, k, k), 0.0, workloads.he_std(c_in, k))
        b = workloads.normal(7102 + 10 * j, (c_out,), 0.0, 0.01) if j % 2 == 0 else None
        ref, sab = oracle.conv2d_f64(x, w, b, s, p)
        data.append((x, w, b, ref, sab))
    plans = []
    for j, (c_in, h, w_, c_out, k, s, p) in enumerate(shapes):
        for v in range(ilpm.num_variants(ilpm.PATH_IGEMM)):
            info = ilpm.variant_info(ilpm.PATH_IGEMM, v)
            if info["k"] != k or info["stride"] != s:
                continue
            for splits in (0, 3, 8):
                try:
                    plan = ilpm.plan_variant(c_in, h, w_, c_out, k, s, p, ilpm.PATH_IGEMM, v, splits)
                except ilpm.IlpmError:
                    continue
                if plan.splits > 1:
                    plans.append((j, plan))
    assert len(plans) >= 8
    # A registered workspace filled with NaN before every call: a partial sum
    # read before the workgroup that wrote it has landed shows as NaN.
    need = max(plan.workspace_bytes for _, plan in plans)
    ws = torch.empty(need // 4 + 64, device="cuda", dtype=torch.float32)
    ilpm.set_workspace(ws)
    try:
        for mode in (ilpm.SPLIT_SUM_KERNEL, ilpm.SPLIT_SUM_FUSED):
            ilpm.set_split_sum(mode)
            outs = []
            # Interleave shapes: plan i of one shape, then one of another.
            for j, plan in plans:
                c_in, h, w_, c_out, k, s, p = shapes[j]
                x, w, b, ref, sab = data[j]
                note(f"[split sum mode {mode}] shape {shapes[j]} {describe(plan)}")
                ws.fill_(float("nan"))
                got = run_conv(x, w, b, s, p, plan=plan)
                ws.fill_(float("nan"))
                relu = ilpm.conv2d_epilogue(dev(x), dev(w), dev(b), s, p, ilpm.EPI_RELU, plan=plan)
                torch.cuda.synchronize()
                outs.append((got, relu.cpu().numpy()))
            if mode == ilpm.SPLIT_SUM_KERNEL:
                base = outs
        for (j, plan), (got, relu), (got0, relu0) in zip(plans, outs, base):
            c_in, _, _, _, k, _, _ = shapes[j]
            np.testing.assert_array_equal(got, got0, err_msg=f"fused vs kernel {describe(plan)}")
            np.testing.assert_array_equal(relu, relu0, err_msg=f"fused relu vs kernel {describe(plan)}")
            np.testing.assert_array_equal(relu, np.maximum(got, 0.0))
            assert_matches(got, data[j][3], data[j][4], c_in, k, f"fused {describe(plan)}")
    finally:
        ilpm.set_split_sum(ilpm.SPLIT_SUM_FUSED)
        torch.cuda.synchronize()
        ilpm.set_workspace(None)


def test_row_kernel_input_layouts(ilpm):
    """The row-segment kernel copies input rows into LDS in 16-byte lanes
    where W is a multiple of 4 and the input is 16-byte aligned, else in
    4-byte lanes: an input 4 bytes off that alignment (a view one float
    into a buffer) gives the same bits, and both match the oracle, on
    strides 1-3, K 1-5, padding on both sides and segments ending past W."""
    torch = torch_cuda()
    shapes = [(3, 20, 36, 40, 3, 2, 1), (1, 9, 64, 20, 5, 1, 2), (2, 11, 44, 64, 3, 3, 1), (1, 8, 16, 17, 5, 2, 2),
              (27, 5, 12, 33, 1, 1, 0), (3, 6, 232, 64, 3, 1, 1)]
    names = {v: ilpm.variant_name(ilpm.PATH_DIRECT, v) for v in range(ilpm.num_variants(ilpm.PATH_DIRECT))}
    rows = [v for v, n in names.items() if n.startswith("direct_rows")]
    for i, (c_in, h, w_, c_out, k, s, p) in enumerate(shapes):
        x, w, b = random_case(4700 + 7 * i, c_in, h, w_, c_out, k, bias=(i % 2 == 0))
        ref, sab = oracle.conv2d_f64(x, w, b, s, p)
        flat = torch.empty(x.size + 1, dtype=torch.float32, device="cuda")
        xm = flat[1:].view(x.shape)
        xm.copy_(torch.from_numpy(x).cuda())
        assert xm.data_ptr() % 16 == 4
        wd, bd = dev(w), dev(b)
        ran = 0
        for v in rows:
            try:
                plan = ilpm.plan_variant(c_in, h, w_, c_out, k, s, p, ilpm.PATH_DIRECT, v)
            except ilpm.IlpmError:
                continue
            note(f"[row layouts {i}] {(c_in, h, w_, c_out, k, s, p)} {describe(plan)}")
            got = run_conv(x, w, b, s, p, plan=plan)
            assert_matches(got, ref, sab, c_in, k, f"rows {i} {names[v]}")
            mis = ilpm.conv2d(xm, wd, bd, s, p, plan=plan)
            torch.cuda.synchronize()
            np.testing.assert_array_equal(mis.cpu().numpy(), got, err_msg=f"rows {i} {names[v]} misaligned input")
            ran += 1
        assert ran, f"no row variant planned {(c_in, h, w_, c_out, k, s, p)}"


def test_low_channel_direct_ragged(ilpm):
    """The low-channel matrix-core direct kernels on ragged shapes: one output
    column or row (W_out = 1 makes the pixel division trivial), planes and
    channel counts that fill no tile, strides 2 and 3, K from 1 to 7 with
    C_in*K*K up to each kernel's limit, bias and none."""
    shapes = [(9, 12, 3, 18, 1, 3, 0), (3, 5, 1, 7, 3, 1, 1), (3, 1, 40, 33, 3, 1, 1), (1, 23, 19, 70, 5, 2, 2),
              (2, 17, 29, 64, 3, 2, 0), (7, 9, 11, 20, 3, 1, 1), (1, 13, 13, 5, 7, 3, 3), (28, 6, 6, 40, 1, 1, 0),
              (3, 224, 37, 64, 3, 1, 1)]
    names = {v: ilpm.variant_name(ilpm.PATH_DIRECT, v) for v in range(ilpm.num_variants(ilpm.PATH_DIRECT))}
    lowc = [v for v, n in names.items() if n.startswith("direct_mfma") or n.startswith("direct_rows")]
    assert any(names[v].startswith("direct_rows") for v in lowc)
    for i, (c_in, h, w_, c_out, k, s, p) in enumerate(shapes):
        x, w, b = random_case(4400 + 7 * i, c_in, h, w_, c_out, k, bias=(i % 2 == 0))
        ref, sab = oracle.conv2d_f64(x, w, b, s, p)
        xi, wi, bi = small_int_case(4500 + 7 * i, c_in, h, w_, c_out, k, bias=(i % 2 == 1))
        refi, _ = oracle.conv2d_f64(xi, wi, bi, s, p)
        first = None
        for v in lowc:
            try:
                plan = ilpm.plan_variant(c_in, h, w_, c_out, k, s, p, ilpm.PATH_DIRECT, v)
            except ilpm.IlpmError:
                continue
            note(f"[lowc {i}] {(c_in, h, w_, c_out, k, s, p)} {describe(plan)}")
            got = run_conv(x, w, b, s, p, plan=plan)
            assert_matches(got, ref, sab, c_in, k, f"lowc {i} v{v}")
            # Every low-channel kernel runs the same matrix-instruction chain
            # (slots k = 4s + g in order from the bias; slots past C_in*K*K
            # add zero products), so they agree bit for bit.
            if first is None:
                first = (names[v], got)
            else:
                np.testing.assert_array_equal(got, first[1], err_msg=f"lowc {i} {names[v]} vs {first[0]}")
            got = run_conv(xi, wi, bi, s, p, plan=plan)
            np.testing.assert_array_equal(got.astype(np.float64), refi, err_msg=f"lowc {i} v{v} small integers")
