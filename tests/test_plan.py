"""Host-side tests of the C-ABI library (no GPU needed): exported symbols,
presets, integer bookkeeping against the oracle's independent plan code, and
error paths."""
import itertools
import re

import pytest

import oracle
from paper_2607_20501_amd import mk, workloads

ROOT_H = __import__("os").path.join(__import__("os").path.dirname(__file__), "..", "include")


def test_library_exports_every_declared_symbol():
    import ctypes
    import os
    lib = ctypes.CDLL(mk.LIB_PATH)
    declared = set()
    for h in os.listdir(ROOT_H):
        if h != "mk.h":
            continue
        text = open(os.path.join(ROOT_H, h)).read()
        declared |= set(re.findall(r"\b(mk_[a-z_]+)\s*\(", text))
    assert declared == set(mk.EXPORTS)
    for name in declared:
        assert hasattr(lib, name), name


def small_modules():
    return [
        workloads.linear_relu_rowsum(M=37, K=70, N=90),
        workloads.gemm_gelu_softmax(M=67, K=96, N=130),
        workloads.conv_relu_gap(N=2, C=5, H=9, W=7, K=6),
        workloads.mlp_block(M=33, D=64, F=96),
        workloads.transformer_layer(B=2, S=40, D=64, H=2, F=96),
    ]


FULL = [workloads.full_size(k) for k in range(1, 6)]

EXPECTED_PRESETS = {
    # split: one subkernel per op, bias / residual joins its contraction
    "split": [[0, 0, 1, 2], [0, 0, 1, 2, 3], [0, 0, 1, 2], [0, 1, 2, 3, 3],
              [0, 1, 2, 3, 4, 5, 6, 6, 7, 8, 9, 10, 10]],
    "fused": [[0, 0, 0, 0], [0, 0, 0, 0, 0], [0, 0, 0, 0], [0, 0, 0, 1, 1],
              [0, 0, 1, 1, 1, 1, 2, 2, 3, 3, 3, 4, 4]],
}


@pytest.mark.parametrize("k", range(5))
def test_presets_match_the_decompositions(k):
    for name in ("split", "fused"):
        assert mk.mk_decomposition_preset(FULL[k], name) == EXPECTED_PRESETS[name][k]
        assert mk.mk_decomposition_preset(small_modules()[k], name) == EXPECTED_PRESETS[name][k]


def groupings(n):
    for cuts in itertools.product([0, 1], repeat=n - 1):
        g = [0]
        for c in cuts:
            g.append(g[-1] + c)
        yield g


FIELDS = ["op_begin", "op_end", "out_value", "out_shape", "out_bytes", "ws_offset", "flops",
          "alg_bytes"]


@pytest.mark.parametrize("k", range(5))
def test_bookkeeping_matches_oracle_for_every_accepted_grouping(k):
    for module in (FULL[k], small_modules()[k]):
        n = len(module["ops"])
        accepted = 0
        for g in groupings(n):
            try:
                h = mk.mk_module_create(module, g)
            except mk.MkError as e:
                assert e.status == 4, str(e)   # MK_E_DECOMP
                continue
            accepted += 1
            try:
                ref = oracle.plan(module, g)
                info = mk.mk_module_info(h)
                assert info["n_subkernels"] == len(ref["groups"])
                assert info["ws_intermediate_bytes"] == ref["ws_intermediate_bytes"]
                assert info["flops"] == ref["flops"]
                assert info["alg_bytes"] == ref["alg_bytes"]
                assert info["ws_bytes"] >= info["ws_intermediate_bytes"]
                for i, rg in enumerate(ref["groups"]):
                    s = mk.mk_subkernel_info(h, i)
                    for f in FIELDS:
                        assert s[f] == rg[f], (g, i, f, s[f], rg[f])
            finally:
                mk.mk_module_destroy(h)
        assert accepted >= 2


def check_all_groupings(module):
    n = len(module["ops"])
    accepted = 0
    for g in groupings(n):
        try:
            h = mk.mk_module_create(module, g)
        except mk.MkError as e:
            assert e.status == 4, str(e)
            continue
        accepted += 1
        try:
            ref = oracle.plan(module, g)
            info = mk.mk_module_info(h)
            assert (info["n_subkernels"], info["flops"], info["alg_bytes"]) == \
                (len(ref["groups"]), ref["flops"], ref["alg_bytes"])
            for i, rg in enumerate(ref["groups"]):
                s = mk.mk_subkernel_info(h, i)
                for f in FIELDS:
                    assert s[f] == rg[f], (g, i, f, s[f], rg[f])
        finally:
            mk.mk_module_destroy(h)
    return accepted


@pytest.mark.parametrize("pool", ["GMP", "LPPOOL"])
def test_pooling_variants_plan_like_gap(pool):
    """Sec. 4's MobileNet adaptation: replacing average pooling by max or LP
    pooling swaps one subkernel.  Every grouping the GAP module accepts is
    accepted with the same bookkeeping, the conv subkernel of the split form
    is unchanged, and the fused form still ends in the conv subkernel."""
    for kw in ({}, dict(N=2, C=5, H=9, W=7, K=6)):
        gap = workloads.conv_relu_gap(**kw)
        var = workloads.conv_relu_gap(pool=pool, p=3.0, **kw)
        assert check_all_groupings(var) == check_all_groupings(gap)
        for dec in ("split", "fused"):
            assert mk.mk_decomposition_preset(var, dec) == mk.mk_decomposition_preset(gap, dec)
        a, b = mk.Module(gap, "split").subkernels(), mk.Module(var, "split").subkernels()
        assert a[:-1] == b[:-1]
        assert b[-1]["family"] == a[-1]["family"] == "ROW"
        assert [s["family"] for s in mk.Module(var, "fused").subkernels()] == ["CONV"]
    with pytest.raises(mk.MkError):
        mk.mk_module_create(workloads.conv_relu_gap(N=1, C=4, H=5, W=5, K=3, pool="LPPOOL",
                                                    p=0.0), [0, 0, 0, 0])


def test_post_ln_block_plans():
    """The CvT post-LN FFN: the split form keeps the LayerNorm as a row
    subkernel; the fused form ends the second GEMM with it (a terminal that
    needs the whole row, like softmax)."""
    for m in (workloads.cvt_ffn_block(), workloads.cvt_ffn_block(M=37, D=100, F=72)):
        assert mk.mk_decomposition_preset(m, "split") == [0, 0, 1, 2, 2, 2, 3]
        assert mk.mk_decomposition_preset(m, "fused") == [0, 0, 0, 1, 1, 1, 1]
        f = mk.Module(m, "fused").subkernels()
        assert [s["family"] for s in f] == ["GEMM", "GEMM"]
        assert f[1]["n_launches"] == 2            # GEMM + LayerNorm finisher
        assert check_all_groupings(m) >= 8


def test_hand_computed_full_size_integers():
    c2 = mk.Module(FULL[1], "fused")
    assert c2.info["flops"] == 2 * 8192 * 4096 * 4096 == 274877906944
    assert c2.info["alg_bytes"] == (8192 * 4096 * 2 + 4096 * 4096 + 4096) * 2
    c4 = mk.Module(FULL[3], "split")
    sk = c4.subkernels()
    assert [s["ws_offset"] for s in sk] == [0, 134217728, 134217728 + 469762048, -1]
    assert c4.info["flops"] == 2 * 2 * 16384 * 4096 * 14336
    c5 = mk.Module(FULL[4], "fused")
    s5 = c5.subkernels()
    assert [s["family"] for s in s5] == ["GEMM", "ATTN", "GEMM", "GEMM", "GEMM"]
    causal = 2 * 2 * 8 * 16 * 128 * (2048 * 2049 // 2)
    assert s5[1]["flops"] == causal
    assert c5.info["flops"] == (2 * 16384 * 2048 * (6144 + 2048 + 8192 + 8192)) + causal


def test_error_paths():
    m = workloads.mlp_block(M=8, D=16, F=32)
    with pytest.raises(mk.MkError) as e:
        mk.mk_module_create(m, [0, 1, 0, 1, 1])
    assert e.value.status == 4
    with pytest.raises(mk.MkError) as e:
        mk.mk_module_create(m, [1, 1, 1, 1, 1])
    assert e.value.status == 4
    # A group that hides a value another group reads.
    t = workloads.transformer_layer(B=1, S=8, D=16, H=2, F=32)
    with pytest.raises(mk.MkError):
        mk.mk_module_create(t, [0] * 13)
    bad = dict(m)
    bad["ops"] = [dict(o) for o in m["ops"]]
    bad["inputs"] = [[8, 16], [16], [16], [32, 17], [16, 32]]
    with pytest.raises(mk.MkError) as e:
        mk.mk_module_create(bad, [0, 1, 2, 3, 3])
    assert e.value.status == 2          # MK_E_SHAPE
    bad2 = dict(m, dtype=7)
    with pytest.raises(mk.MkError) as e:
        mk.mk_module_create(bad2, [0, 1, 2, 3, 3])
    assert e.value.status == 3          # MK_E_DTYPE
    bad3 = dict(m)
    bad3["ops"] = [dict(o) for o in m["ops"]]
    bad3["ops"][0] = dict(bad3["ops"][0], **{"in": [9, 1, 2]})
    with pytest.raises(mk.MkError) as e:
        mk.mk_module_create(bad3, [0, 1, 2, 3, 3])
    assert e.value.status == 1          # MK_E_INVALID_ARG
    h = mk.Module(m, "split")
    with pytest.raises(mk.MkError) as e:
        h.select(0, 55)
    assert e.value.status == 5          # MK_E_UNSUPPORTED
    with pytest.raises(mk.MkError) as e:
        h.select(9, 0)
    assert e.value.status == 1
    # Workspace too small: rejected before any device work.
    with pytest.raises(mk.MkError) as e:
        mk.mk_run(h.h, [1, 2, 3, 4, 5], 6, 7, 0, None)
    assert e.value.status == 6          # MK_E_WORKSPACE
    with pytest.raises(mk.MkError) as e:
        mk.mk_run(h.h, [1, 0, 3, 4, 5], 6, 7, 1 << 40, None)
    assert e.value.status == 1


def test_swap_keeps_workspace_and_reports_impl():
    m = mk.Module(workloads.gemm_gelu_softmax(M=64, K=64, N=512), "fused")
    ws = m.workspace_size()
    m.select(0, mk.IMPL_SIMPLE)
    assert m.subkernels()[0]["impl"] == mk.IMPL_SIMPLE
    assert m.workspace_size() == ws
    assert m.subkernels()[0]["scratch_bytes"] <= ws
    assert m.subkernels()[0]["n_launches"] == 2


def test_empty_dimensions_are_rejected_by_both_sides():
    """A zero-sized dimension is an error (MK_E_SHAPE) in the library and in
    the oracle alike; there is no empty launch to take."""
    for M in (0,):
        m = workloads.linear_relu_rowsum(M=M, K=8, N=8)
        with pytest.raises(mk.MkError) as e:
            mk.mk_module_create(m, [0, 0, 0, 0])
        assert e.value.status == 2            # MK_E_SHAPE
        with pytest.raises(ValueError):
            oracle.plan(m, [0, 0, 0, 0])
    m = workloads.conv_relu_gap(N=1, C=4, H=0, W=5, K=3)
    with pytest.raises(mk.MkError):
        mk.mk_module_create(m, [0, 0, 0, 0])


def test_tuned_limit_is_reported_and_strict_mode_raises():
    """The tuned implementation names why it runs the simple kernels
    (mk_tuned_limit), the binding warns about it, and strict=True refuses."""
    cases = [
        (workloads.linear_relu_rowsum(M=64, K=256, N=128, dtype="bf16"), [0, 0, 0, 0],
         {0: "none"}),
        (workloads.linear_relu_rowsum(M=64, K=250, N=128, dtype="bf16"), [0, 0, 0, 0],
         {0: "align"}),   # K not a multiple of 8 bf16
        (workloads.linear_relu_rowsum(M=64, K=126, N=128, dtype="f32"), [0, 0, 0, 0],
         {0: "align"}),   # K not a multiple of 4 fp32
        (workloads.gemm_gelu_softmax(M=64, K=64, N=100, dtype="bf16"), [0, 0, 0, 0, 0],
         {0: "align"}),   # [K, N] weight with N not a multiple of 8
        (workloads.conv_relu_gap(N=2, C=5, H=9, W=7, K=6), [0, 0, 0, 0], {0: "shape"}),
        (workloads.conv_relu_gap(N=2, C=64, H=16, W=16, K=32), [0, 0, 0, 0], {0: "none"}),
        (workloads.conv_relu_gap(N=2, C=64, H=8, W=8, K=32), [0, 0, 0, 0],
         {0: "shape"}),   # pooled 8 x 8 image smaller than a column tile
        (workloads.causal_attention_block(B=1, S=64, D=128, H=2, dtype="bf16"),
         [0, 1, 1, 1, 1, 2], {0: "none", 1: "none", 2: "none"}),
        (workloads.causal_attention_block(B=1, S=64, D=128, H=2, dtype="f32"),
         [0, 1, 1, 1, 1, 2], {0: "none", 1: "dtype", 2: "none"}),
        (workloads.causal_attention_block(B=1, S=64, D=128, H=4, dtype="bf16"),
         [0, 1, 1, 1, 1, 2], {0: "none", 1: "shape", 2: "none"}),   # head dim 32
    ]
    for module, groups, want in cases:
        with __import__("warnings").catch_warnings(record=True) as w:
            __import__("warnings").simplefilter("always")
            m = mk.Module(module, groups)
        got = {i: s["tuned_limit"] for i, s in enumerate(m.subkernels())}
        assert got == want, module["name"]
        limited = any(v != "none" for v in want.values())
        assert any(issubclass(x.category, mk.TunedLimitWarning) for x in w) == limited
        if limited:
            with pytest.raises(mk.MkError) as e:
                mk.Module(module, groups, strict=True)
            assert e.value.status == 5          # MK_E_UNSUPPORTED
        else:
            mk.Module(module, groups, strict=True)
        m.select(0, mk.IMPL_SIMPLE)               # reported whichever impl is selected
        assert m.subkernels()[0]["tuned_limit"] == want[0]
    for k in range(1, 6):                         # every full-size workload runs tuned
        full = workloads.full_size(k)
        for preset in ("split", "fused"):
            mk.Module(full, preset, strict=True)


def test_profile_launch_index_is_checked_before_any_device_call():
    m = mk.Module(workloads.gemm_gelu_softmax(M=64, K=64, N=512), "fused")
    for bad in (-2, m.launches_per_run()):
        with pytest.raises(mk.MkError) as e:
            m.profile_begin(4, only_launch=bad)
        assert e.value.status == 1            # MK_E_INVALID_ARG
