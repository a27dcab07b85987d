"""The C ABI on the host: the library loads, exports every declared symbol, and
its pure-host entry points (validation, planning, workspace sizing, status
text) behave as include/ilpm.h states.  No kernel is launched."""
import ctypes
import os
import re

import pytest

import paper_1909_02765_amd as ilpm
import workloads

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "ilpm.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(ilpm_\w+)\s*\(", text)))


def test_every_declared_symbol_is_exported():
    names = declared_functions()
    assert len(names) >= 12
    for n in names:
        assert hasattr(ilpm.lib, n), f"{n} declared in ilpm.h but not exported"


def test_status_strings():
    assert ilpm.status_str(0) == "ok"
    seen = set()
    for code in (-1, -2, -3, -4, -5):
        s = ilpm.status_str(code)
        assert s and s != "unknown status"
        seen.add(s)
    assert len(seen) == 5
    assert ilpm.status_str(7) == "unknown status"


def _validate(inp=0x1000, w=0x100000, b=None, c_in=3, h=8, wd=8, c_out=4, k=3, s=1, p=1, out=0x200000):
    return ilpm.lib.ilpm_conv2d_validate(inp, w, b, c_in, h, wd, c_out, k, s, p, out)


def test_validate_ok():
    assert _validate() == ilpm.OK
    assert _validate(b=0x300000) == ilpm.OK


@pytest.mark.parametrize("kw", [
    dict(inp=None), dict(w=None), dict(out=None),
    dict(c_in=0), dict(h=0), dict(wd=-1), dict(c_out=0), dict(k=0), dict(s=0), dict(s=-2), dict(p=-1),
    dict(h=2, k=5, p=1),          # H_out < 1
    dict(wd=1, k=3, p=0),         # W_out < 1
    dict(out=0x1000 + 16),        # out overlaps the input
    dict(out=0x100000 + 4),       # out overlaps the weights
    dict(b=0x200000 + 8),         # out overlaps the bias
    dict(inp=0x1002),             # misaligned
])
def test_validate_invalid(kw):
    assert _validate(**kw) == ilpm.ERR_INVALID_ARG


def test_validate_unsupported_size():
    # 2^31 input elements
    assert _validate(c_in=2, h=32768, wd=32768, out=0x7000000000000) == ilpm.ERR_UNSUPPORTED


def test_fwd_rejects_before_any_launch():
    # Returns from the argument check without touching a device.
    rc = ilpm.lib.ilpm_conv2d_fwd(None, 0x1000, None, 3, 8, 8, 4, 3, 1, 1, 0x100000, None)
    assert rc == ilpm.ERR_INVALID_ARG
    rc = ilpm.lib.ilpm_conv2d_fwd(0x1000, 0x100000, None, 3, 2, 2, 4, 5, 1, 0, 0x200000, None)
    assert rc == ilpm.ERR_INVALID_ARG
    rc = ilpm.lib.ilpm_maxpool2x2(0x1000, 3, 1, 8, 0x2000, None)
    assert rc == ilpm.ERR_INVALID_ARG
    rc = ilpm.lib.ilpm_relu_inplace(None, 10, None)
    assert rc == ilpm.ERR_INVALID_ARG


def test_set_workspace_rejects_misaligned():
    assert ilpm.lib.ilpm_set_workspace(ctypes.c_void_p(0x1000 + 16), 4096, None) == ilpm.ERR_INVALID_ARG


def test_variants_table():
    nd = ilpm.num_variants(ilpm.PATH_DIRECT)
    assert nd >= 3
    assert [ilpm.variant_name(ilpm.PATH_DIRECT, v) for v in (0, 1)] == ["direct_lds_t8x32_co16", "direct_global"]
    n = ilpm.num_variants(ilpm.PATH_IGEMM)
    assert n >= 4
    assert ilpm.num_variants(7) == 0
    ks = set()
    for v in range(n):
        info = ilpm.variant_info(ilpm.PATH_IGEMM, v)
        assert info["co_tile"] % 16 == 0 and info["tile_h"] >= 1 and info["tile_w"] >= 1
        ks.add((info["k"], info["stride"]))
    assert {(3, 1), (3, 2), (1, 1), (5, 1)} <= ks
    with pytest.raises(ilpm.IlpmError):
        ilpm.variant_info(ilpm.PATH_IGEMM, n)


@pytest.mark.parametrize("case", workloads.ALL_CASES, ids=lambda c: c.name)
def test_plan_for_every_workload(case):
    d = case.dims()
    p = ilpm.plan(d["c_in"], d["h"], d["w"], d["c_out"], d["k"], d["stride"], d["pad"])
    assert p.h_out == ilpm.out_size(d["h"], d["k"], d["stride"], d["pad"])
    assert p.w_out == ilpm.out_size(d["w"], d["k"], d["stride"], d["pad"])
    assert p.grid >= 1 and p.block in (64, 128, 256, 512, 768, 1024)
    assert p.lds_bytes <= 160 * 1024
    if p.splits > 1:
        assert p.workspace_bytes > 0
    assert ilpm.workspace_size(d["c_in"], d["h"], d["w"], d["c_out"], d["k"], d["stride"], d["pad"]) \
        == p.workspace_bytes


def test_plan_variant_rules():
    # A 3x3/stride-1 variant refuses a 5x5 filter; direct variants take any.
    v33 = next(v for v in range(ilpm.num_variants(ilpm.PATH_IGEMM))
               if ilpm.variant_info(ilpm.PATH_IGEMM, v)["k"] == 3
               and ilpm.variant_info(ilpm.PATH_IGEMM, v)["stride"] == 1)
    with pytest.raises(ilpm.IlpmError):
        ilpm.plan_variant(8, 7, 7, 16, 5, 1, 2, ilpm.PATH_IGEMM, v33)
    p = ilpm.plan_variant(8, 7, 7, 16, 7, 3, 2, ilpm.PATH_DIRECT, 0)
    assert p.path == ilpm.PATH_DIRECT and p.h_out == 2
    p = ilpm.plan_variant(512, 14, 14, 512, 3, 1, 1, ilpm.PATH_IGEMM, v33, 4)
    assert p.splits == 4 and p.workspace_bytes > 0
    # more splits than input-channel stages is refused
    with pytest.raises(ilpm.IlpmError):
        ilpm.plan_variant(8, 14, 14, 64, 3, 1, 1, ilpm.PATH_IGEMM, v33, 2)


def test_fixed_stage_variants_plan_whole_splits():
    """A three-buffer variant is built for an exact stage count: it plans a
    shape only in splits of exactly that many channel chunks."""
    fixed = [v for v in range(ilpm.num_variants(ilpm.PATH_IGEMM))
             if ilpm.variant_info(ilpm.PATH_IGEMM, v)["stages"]]
    assert fixed
    for v in fixed:
        info = ilpm.variant_info(ilpm.PATH_IGEMM, v)
        k, s, ns, cc = info["k"], info["stride"], info["stages"], info["ci_chunk"]
        for splits in (1, 2, 3):
            c_in = ns * cc * splits - cc // 2  # the last chunk half full
            p = ilpm.plan_variant(c_in, 20, 20, 40, k, s, k // 2, ilpm.PATH_IGEMM, v)
            assert p.splits == splits
            p = ilpm.plan_variant(c_in, 20, 20, 40, k, s, k // 2, ilpm.PATH_IGEMM, v, splits)
            assert p.splits == splits
            with pytest.raises(ilpm.IlpmError):
                ilpm.plan_variant(c_in, 20, 20, 40, k, s, k // 2, ilpm.PATH_IGEMM, v, splits + 1)
        with pytest.raises(ilpm.IlpmError):  # one chunk more than a whole number of splits
            ilpm.plan_variant(ns * cc + 1, 20, 20, 40, k, s, k // 2, ilpm.PATH_IGEMM, v)
    for v in range(ilpm.num_variants(ilpm.PATH_DIRECT)):
        info = ilpm.variant_info(ilpm.PATH_DIRECT, v)
        assert info["stages"] == 0 and info["buffers"] == 0 and not info["weights_lds"]
    for v in range(ilpm.num_variants(ilpm.PATH_IGEMM)):
        info = ilpm.variant_info(ilpm.PATH_IGEMM, v)
        assert (info["buffers"] > 2) == (info["stages"] > 0)
        assert info["ci_chunk"] > 0 and info["buffers"] >= 2


def test_progressive_first_stage_plans_two_stages_per_split():
    """A variant with a progressive first stage computes that stage from
    buffers of its own and goes on to a second: it plans only splits of at
    least two channel chunks, and its automatic split count keeps that."""
    pf = [v for v in range(ilpm.num_variants(ilpm.PATH_IGEMM))
          if ilpm.variant_info(ilpm.PATH_IGEMM, v)["progressive_first"]]
    assert pf
    for v in pf:
        info = ilpm.variant_info(ilpm.PATH_IGEMM, v)
        k, s, cc = info["k"], info["stride"], info["ci_chunk"]
        assert info["stages"] == 0 and info["buffers"] == 2 and not info["weights_lds"]
        with pytest.raises(ilpm.IlpmError):  # one chunk
            ilpm.plan_variant(cc, 20, 20, 40, k, s, k // 2, ilpm.PATH_IGEMM, v, 1)
        assert ilpm.plan_variant(cc + 1, 20, 20, 40, k, s, k // 2, ilpm.PATH_IGEMM, v, 1).splits == 1
        with pytest.raises(ilpm.IlpmError):  # 3 chunks in 2 splits leaves a split of one
            ilpm.plan_variant(3 * cc, 20, 20, 40, k, s, k // 2, ilpm.PATH_IGEMM, v, 2)
        assert ilpm.plan_variant(4 * cc, 20, 20, 40, k, s, k // 2, ilpm.PATH_IGEMM, v, 2).splits == 2
        for c_in in (2 * cc, 5 * cc - 1, 16 * cc):  # few output tiles: the automatic count splits
            p = ilpm.plan_variant(c_in, 14, 14, 40, k, s, k // 2, ilpm.PATH_IGEMM, v)
            nchunks = -(-c_in // cc)
            cps = -(-nchunks // p.splits)
            assert cps >= 2 and nchunks - (p.splits - 1) * cps >= 2


_PLAN_IN_CHILD = r"""
import json, sys
sys.path.insert(0, {root!r})
import paper_1909_02765_amd as ilpm
out = []
for shape in {shapes!r}:
    try:
        p = ilpm.plan(*shape)
        out.append(dict(path=p.path, tile=[p.tile_h, p.tile_w], splits=p.splits,
                        name=ilpm.variant_name(p.path, p.variant)))
    except ilpm.IlpmError as e:
        out.append(dict(status=e.status))
print(json.dumps(out))
"""


def plans_with_env(env_extra, shapes):
    """The default plans of `shapes` in a fresh process whose environment has
    env_extra (the library reads its overrides once, at its first plan)."""
    import json
    import subprocess
    import sys
    env = {k: v for k, v in os.environ.items() if not k.startswith("ILPM_")}
    env.update(env_extra)
    r = subprocess.run([sys.executable, "-c", _PLAN_IN_CHILD.format(root=ROOT, shapes=shapes)],
                       capture_output=True, text=True, env=env, timeout=300)
    assert r.returncode == 0, r.stderr
    return json.loads(r.stdout.strip().splitlines()[-1])


CONV2X = (64, 56, 56, 64, 3, 1, 1)
CONV4X = (256, 14, 14, 256, 3, 1, 1)


def test_plan_env_force_path():
    base, forced = plans_with_env({}, [CONV2X]), plans_with_env({"ILPM_FORCE_PATH": "direct"}, [CONV2X])
    assert base[0]["path"] == ilpm.PATH_IGEMM
    assert forced[0]["path"] == ilpm.PATH_DIRECT
    assert plans_with_env({"ILPM_FORCE_PATH": "gemm"}, [CONV2X])[0]["path"] == ilpm.PATH_IGEMM


def test_plan_env_tile_override():
    """ILPM_TILE=<h>x<w> keeps only variants with that output tile; a tile no
    variant has makes planning fail with ILPM_ERR_UNSUPPORTED."""
    got = plans_with_env({"ILPM_TILE": "7x7"}, [CONV4X, CONV2X])
    assert all(g["tile"] == [7, 7] for g in got), got
    got = plans_with_env({"ILPM_TILE": "4x4"}, [CONV4X])
    assert got[0]["tile"] == [4, 4], got
    got = plans_with_env({"ILPM_TILE": "1x1"}, [CONV4X])  # only the global-memory direct kernel
    assert got[0]["path"] == ilpm.PATH_DIRECT and got[0]["tile"] == [1, 1], got
    got = plans_with_env({"ILPM_TILE": "3x5"}, [CONV4X])
    assert got[0] == {"status": ilpm.ERR_UNSUPPORTED}, got
    got = plans_with_env({"ILPM_TILE": "1x1", "ILPM_FORCE_PATH": "igemm"}, [CONV4X])
    assert got[0] == {"status": ilpm.ERR_UNSUPPORTED}, got


def test_plan_env_split_override():
    got = plans_with_env({"ILPM_SPLIT": "2", "ILPM_TILE": "7x7"}, [CONV4X])
    assert got[0]["splits"] == 2 and got[0]["tile"] == [7, 7], got


def test_plan_is_stable_across_calls():
    a, b = ilpm.plan(*CONV4X), ilpm.plan(*CONV4X)
    assert a.as_dict() == b.as_dict()


@pytest.mark.parametrize("name,want", [
    (b"gfx950", ilpm.OK), (b"gfx950:sramecc+:xnack-", ilpm.OK), (b"gfx950:xnack+", ilpm.OK),
    (b"gfx942", ilpm.ERR_ARCH), (b"gfx942:sramecc+:xnack-", ilpm.ERR_ARCH), (b"gfx90a", ilpm.ERR_ARCH),
    (b"gfx9501", ilpm.ERR_ARCH), (b"gfx95", ilpm.ERR_ARCH), (b"", ilpm.ERR_ARCH), (b"gfx1201", ilpm.ERR_ARCH),
    (None, ilpm.ERR_INVALID_ARG)])
def test_arch_check(name, want):
    """The architecture check behind ILPM_ERR_ARCH: gfx950 with any feature
    suffix passes, every other name (including a longer one that starts with
    gfx950) is refused."""
    assert ilpm.lib.ilpm_arch_supported(name) == want
    if want == ilpm.ERR_ARCH:
        assert ilpm.status_str(want) == "device is not gfx950"


def test_fwd_plan_rejects_foreign_plan():
    p = ilpm.plan(64, 56, 56, 64, 3, 1, 1)
    rc = ilpm.lib.ilpm_conv2d_fwd_plan(0x1000, 0x10000000, None, 64, 28, 28, 64, 3, 1, 1, 0x20000000,
                                       ctypes.byref(p), None)
    assert rc == ilpm.ERR_INVALID_ARG


def test_tuned_table_entries_resolve():
    """Every entry of the compiled-in tuning table names a variant that exists
    and accepts its shape, and the default plan for that shape is that entry."""
    import re
    inc = os.path.join(ROOT, "paper_1909_02765_amd", "csrc", "tuned_plans.inc")
    rows = re.findall(r'\{(\d+), (\d+), (\d+), (\d+), (\d+), (\d+), (\d+), "([^"]*)", (\d+)\}', open(inc).read())
    names = {(path, ilpm.variant_name(path, v)): v for path in (0, 1) for v in range(ilpm.num_variants(path))}
    n = 0
    for r in rows:
        c_in, h, w, c_out, k, s, p = map(int, r[:7])
        if c_in == 0:
            continue
        name, splits = r[7], int(r[8])
        path = 1 if (1, name) in names else 0
        assert (path, name) in names, f"unknown variant {name}"
        plan = ilpm.plan(c_in, h, w, c_out, k, s, p)
        assert plan.path == path and ilpm.variant_name(plan.path, plan.variant) == name
        if path == 1:
            assert plan.splits == splits
        n += 1
    assert n >= 10


def test_prepacked_size():
    """Packed weights of a matrix-core plan are padded to whole output-channel
    tiles and input-channel chunks; a direct plan's are an OIHW copy."""
    import ctypes
    for (c_in, c_out, k, s) in [(64, 64, 3, 1), (13, 40, 3, 1), (512, 512, 5, 1), (37, 70, 1, 1), (128, 256, 3, 2)]:
        for v in range(ilpm.num_variants(ilpm.PATH_IGEMM)):
            info = ilpm.variant_info(ilpm.PATH_IGEMM, v)
            if info["k"] != k or info["stride"] != s:
                continue
            ci = c_in
            if info["stages"]:  # a fixed-stage variant: a channel count it takes, last chunk partial
                ci = info["stages"] * info["ci_chunk"] - 3
            if info["progressive_first"]:  # at least two stages, the last partial
                ci = max(ci, 2 * info["ci_chunk"] - 3)
            if info["consecutive_channels"]:  # C_in a multiple of 4, the last chunk partial
                ci = -(-ci // 4) * 4
            p = ilpm.plan_variant(ci, 16, 16, c_out, k, s, k // 2, ilpm.PATH_IGEMM, v, 0 if info["stages"] else 1)
            cot, cc = p.co_tile, p.ci_chunk
            want = -(-c_out // cot) * cot * (-(-ci // cc) * cc) * k * k * 4
            if info["weights_lds"]:  # such a variant reads OIHW; its prepacked weights are a copy
                want = c_out * ci * k * k * 4
            assert ilpm.prepacked_size(p, ci, c_out, k) == want
            with pytest.raises(ilpm.IlpmError):
                ilpm.prepacked_size(p, ci, c_out, k + 2)
    p = ilpm.plan_variant(3, 16, 16, 8, 7, 1, 3, ilpm.PATH_DIRECT, 0)
    assert ilpm.prepacked_size(p, 3, 8, 7) == 8 * 3 * 49 * 4


def test_prepacked_rejects_before_any_launch():
    import ctypes
    p = ilpm.plan(64, 56, 56, 64, 3, 1, 1)
    lib = ilpm.lib
    assert lib.ilpm_conv2d_prepack_weights(None, 64, 64, 3, ctypes.byref(p), 0x100000, None) == ilpm.ERR_INVALID_ARG
    assert lib.ilpm_conv2d_prepack_weights(0x1000 + 4, 64, 64, 3, ctypes.byref(p), 0x100000, None) \
        == ilpm.ERR_INVALID_ARG                                        # misaligned
    assert lib.ilpm_conv2d_prepack_weights(0x1000, 64, 64, 5, ctypes.byref(p), 0x100000, None) \
        == ilpm.ERR_INVALID_ARG                                        # K the plan does not take
    assert lib.ilpm_conv2d_prepack_weights(0x1000, 64, 64, 3, ctypes.byref(p), 0x1000 + 256, None) \
        == ilpm.ERR_INVALID_ARG                                        # overlap
    # a plan for another shape is refused
    assert lib.ilpm_conv2d_fwd_prepacked(0x1000, 0x10000000, None, 64, 28, 28, 64, 3, 1, 1, ctypes.byref(p),
                                         0x20000000, None) == ilpm.ERR_INVALID_ARG
    assert lib.ilpm_conv2d_fwd_prepacked(0x1000, None, None, 64, 56, 56, 64, 3, 1, 1, ctypes.byref(p),
                                         0x20000000, None) == ilpm.ERR_INVALID_ARG


def test_epilogue_argument_checks():
    lib = ilpm.lib
    # unknown epilogue bits
    assert lib.ilpm_conv2d_fwd_epilogue(0x1000, 0x100000, None, 3, 8, 8, 4, 3, 1, 1, 4, None, 0x200000, None) \
        == ilpm.ERR_INVALID_ARG
    # pooling needs a 2x2 window: H_out = 1
    assert lib.ilpm_conv2d_fwd_epilogue(0x1000, 0x100000, None, 3, 1, 8, 4, 1, 1, 0, ilpm.EPI_MAXPOOL2, None,
                                        0x200000, None) == ilpm.ERR_INVALID_ARG
    # the pooled output is a quarter of the conv output: placing it right after
    # the input is fine for the overlap check, one float earlier is not
    in_b = 4 * 3 * 8 * 8
    assert lib.ilpm_conv2d_validate(0x1000, 0x100000, None, 3, 8, 8, 4, 3, 1, 1, 0x1000 + in_b) == ilpm.OK
    assert lib.ilpm_conv2d_fwd_epilogue(0x1000, 0x100000, None, 3, 8, 8, 4, 3, 1, 1, ilpm.EPI_MAXPOOL2, None,
                                        0x1000 + in_b - 4, None) == ilpm.ERR_INVALID_ARG


def test_epilogue_workspace_size():
    # pooling keeps the full-size convolution output (times the splits) in the workspace
    for shape in [(64, 56, 56, 64, 3, 1, 1), (512, 7, 7, 512, 3, 1, 1), (3, 224, 224, 64, 3, 1, 1)]:
        c_in, h, w, c_out, k, s, p = shape
        plan = ilpm.plan(*shape)
        full = 4 * c_out * ilpm.out_size(h, k, s, p) * ilpm.out_size(w, k, s, p)
        assert ilpm.epilogue_workspace_size(*shape, 0) == plan.workspace_bytes
        assert ilpm.epilogue_workspace_size(*shape, ilpm.EPI_RELU) == plan.workspace_bytes
        assert ilpm.epilogue_workspace_size(*shape, ilpm.EPI_MAXPOOL2) == full * max(plan.splits, 1)


def test_winograd_sizes_and_argument_checks():
    import ctypes
    n = ctypes.c_size_t()
    assert ilpm.lib.ilpm_winograd_filter_size(64, 128, ctypes.byref(n)) == ilpm.OK and n.value == 16 * 64 * 128 * 4
    assert ilpm.lib.ilpm_winograd_filter_size(0, 128, ctypes.byref(n)) == ilpm.ERR_INVALID_ARG
    assert ilpm.lib.ilpm_conv2d_winograd_workspace_size(64, 224, 224, 64, 1, ctypes.byref(n)) == ilpm.OK
    assert n.value == 4 * 16 * (64 + 64) * 112 * 112
    # odd output: 9x11 with pad 1 -> 5x6 tiles
    assert ilpm.lib.ilpm_conv2d_winograd_workspace_size(3, 9, 11, 2, 1, ctypes.byref(n)) == ilpm.OK
    assert n.value == 4 * 16 * (3 + 2) * 5 * 6
    lib = ilpm.lib
    assert lib.ilpm_conv2d_fwd_winograd(None, 0x100000, None, 3, 8, 8, 4, 1, 0x200000, None) == ilpm.ERR_INVALID_ARG
    assert lib.ilpm_conv2d_fwd_winograd(0x1002, 0x100000, None, 3, 8, 8, 4, 1, 0x200000, None) == ilpm.ERR_INVALID_ARG
    assert lib.ilpm_conv2d_fwd_winograd(0x1000, 0x100000, None, 3, 1, 8, 4, 0, 0x200000, None) == ilpm.ERR_INVALID_ARG
    assert lib.ilpm_winograd_transform_filter(0x1000, 3, 4, 0x1000 + 64, None) == ilpm.ERR_INVALID_ARG  # overlap


def test_split_sum_mode_switch():
    """The two split-sum modes are accepted (host only, no launch); any other is refused."""
    try:
        assert ilpm.lib.ilpm_set_split_sum(ilpm.SPLIT_SUM_KERNEL) == ilpm.OK
        assert ilpm.lib.ilpm_set_split_sum(ilpm.SPLIT_SUM_FUSED) == ilpm.OK
        for bad in (-1, 2, 99):
            assert ilpm.lib.ilpm_set_split_sum(bad) == ilpm.ERR_INVALID_ARG
            with pytest.raises(ilpm.IlpmError):
                ilpm.set_split_sum(bad)
    finally:
        ilpm.set_split_sum(ilpm.SPLIT_SUM_FUSED)


def test_low_channel_direct_variants_plan_only_short_contractions():
    """The low-channel matrix-core direct kernels take a shape only when the
    whole C_in*K*K contraction fits their one chain of matrix instructions."""
    lowc = [v for v in range(ilpm.num_variants(ilpm.PATH_DIRECT))
            if ilpm.variant_name(ilpm.PATH_DIRECT, v).startswith("direct_mfma_k28")]
    assert lowc
    for v in lowc:
        p = ilpm.plan_variant(3, 224, 224, 64, 3, 1, 1, ilpm.PATH_DIRECT, v)   # 27 products
        info = ilpm.variant_info(ilpm.PATH_DIRECT, v)
        units = -(-64 // info["co_tile"]) * -(-224 * 224 // info["tile_w"])
        assert p.grid == -(-units // 4) and p.block == 256 and p.lds_bytes == 0 and p.workspace_bytes == 0
        with pytest.raises(ilpm.IlpmError):
            ilpm.plan_variant(4, 224, 224, 64, 3, 1, 1, ilpm.PATH_DIRECT, v)  # 36 > 28
    rows = [v for v in range(ilpm.num_variants(ilpm.PATH_DIRECT))
            if ilpm.variant_name(ilpm.PATH_DIRECT, v).startswith("direct_rows_k28")]
    assert rows
    for v in rows:
        # One workgroup per (output row, row segment, channel group); LDS
        # holds the C_in*K input rows the segment reads and one zero row,
        # each padded to whole 256-word DMA chunks of 16-byte lanes (W = 224
        # is a multiple of 4; the copy starts up to 3 columns early), then
        # the group's weights (whole 256-word DMAs) and 64 words of biases.
        p = ilpm.plan_variant(3, 224, 224, 64, 3, 1, 1, ilpm.PATH_DIRECT, v)
        info = ilpm.variant_info(ilpm.PATH_DIRECT, v)
        segs, groups = -(-224 // info["tile_w"]), -(-64 // info["co_tile"])
        lwp = 256 * -(-(info["tile_w"] - 1 + 3 + 3) // 256)
        wregion = 256 * -(-(info["co_tile"] * 27) // 256)
        assert p.grid == 224 * segs * groups and p.block == 256 and p.workspace_bytes == 0
        assert p.lds_bytes == 4 * ((3 * 3 + 1) * lwp + wregion + 64)
        with pytest.raises(ilpm.IlpmError):
            ilpm.plan_variant(4, 224, 224, 64, 3, 1, 1, ilpm.PATH_DIRECT, v)  # 36 > 28
        # W not a multiple of 4: rows of whole 64-word chunks of 4-byte lanes.
        q = ilpm.plan_variant(3, 30, 222, 64, 3, 1, 1, ilpm.PATH_DIRECT, v)
        lwp4 = 64 * -(-(info["tile_w"] - 1 + 3) // 64)
        assert q.lds_bytes == 4 * ((3 * 3 + 1) * lwp4 + wregion + 64)
    big = [v for v in range(ilpm.num_variants(ilpm.PATH_DIRECT))
           if ilpm.variant_name(ilpm.PATH_DIRECT, v).startswith("direct_mfma_k64")]
    for v in big:
        ilpm.plan_variant(7, 30, 30, 20, 3, 2, 1, ilpm.PATH_DIRECT, v)        # 63
        with pytest.raises(ilpm.IlpmError):
            ilpm.plan_variant(8, 30, 30, 20, 3, 1, 1, ilpm.PATH_DIRECT, v)    # 72 > 64


def test_launcher_object_keeps_and_reports():
    """The launcher object behind conv2d_launcher & co.: it holds what it is
    given to keep, passes the marshalled arguments, and turns a non-OK
    status into IlpmError (host only: a stand-in entry point)."""
    import gc
    import weakref

    class Held:
        pass

    calls = []
    held = Held()
    ref = weakref.ref(held)
    ok = ilpm._Launcher(lambda *a: calls.append(a) or ilpm.OK, (1, 2), (held,), "stand_in")
    del held
    gc.collect()
    assert ref() is not None
    ok()
    assert calls == [(1, 2)]
    bad = ilpm._Launcher(lambda *a: ilpm.ERR_INVALID_ARG, (), (), "stand_in")
    with pytest.raises(ilpm.IlpmError):
        bad()
    del ok
    gc.collect()
    assert ref() is None


def test_plan_for_layouts_and_epilogues():
    """ilpm_conv2d_plan_for: no epilogue / OIHW is ilpm_conv2d_plan, prepacked is
    ilpm_conv2d_plan_prepacked; a pooled epilogue takes the pooled table's
    plan (VGG conv4_3: 512->512 at 28x28), ReLU alone does not; bad epilogue
    bits or layouts are refused (host only)."""
    shape = (512, 28, 28, 512, 3, 1, 1)
    same = lambda a, b: a.as_dict() == b.as_dict()
    assert same(ilpm.plan_for(*shape), ilpm.plan(*shape))
    assert same(ilpm.plan_for(*shape, prepacked=True), ilpm.plan_prepacked(*shape))
    assert same(ilpm.plan_for(*shape, epilogue=ilpm.EPI_RELU), ilpm.plan(*shape))
    pooled = ilpm.plan_for(*shape, epilogue=ilpm.EPI_RELU | ilpm.EPI_MAXPOOL2)
    tables = {}
    for name in ("tuned_plans_pooled.inc",):
        for line in open(os.path.join(os.path.dirname(ilpm.__file__), "csrc", name)):
            if line.startswith("{512, 28, 28, 512, 3, 1, 1,"):
                tables[name] = line.split('"')[1], int(line.split('"')[2].strip(" ,}").split("}")[0])
    variant, splits = tables["tuned_plans_pooled.inc"]
    assert ilpm.variant_name(pooled.path, pooled.variant) == variant and pooled.splits == splits
    out = ilpm.ilpm_plan()
    for epi, packed in ((4, 0), (0, 2), (0, -1)):
        assert ilpm.lib.ilpm_conv2d_plan_for(*shape, epi, packed, ctypes.byref(out)) == ilpm.ERR_INVALID_ARG


def test_consecutive_channel_variants_need_c_in_multiple_of_4():
    """The 1x1 variants whose lanes take four consecutive input channels per
    16-byte weight load plan only for C_in a multiple of 4 (a load then never
    reaches past the weight tensor); the other 1x1 variant takes any C_in."""
    names = {ilpm.variant_name(ilpm.PATH_IGEMM, v): v for v in range(ilpm.num_variants(ilpm.PATH_IGEMM))}
    c1 = {n for n, v in names.items() if ilpm.variant_info(ilpm.PATH_IGEMM, v)["consecutive_channels"]}
    assert c1 == {"k1s1_t7x7_co64", "k1s1_t14x14_co64", "k1s1_t4x4_co16_k4"}
    for name in sorted(c1):
        v = names[name]
        for c_in in (4, 8, 36, 512):
            ilpm.plan_variant(c_in, 7, 7, 64, 1, 1, 0, ilpm.PATH_IGEMM, v, 1)
        for c_in in (1, 6, 37, 513):
            with pytest.raises(ilpm.IlpmError):
                ilpm.plan_variant(c_in, 7, 7, 64, 1, 1, 0, ilpm.PATH_IGEMM, v, 1)
    for c_in in (1, 6, 37, 513):
        ilpm.plan_variant(c_in, 7, 7, 64, 1, 1, 0, ilpm.PATH_IGEMM, names["k1s1_t7x7_co64_k4"], 1)
