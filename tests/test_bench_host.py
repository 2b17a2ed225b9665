"""Host-side accounting of bench.py (no GPU): kernel-name handling, the op
rates against the MI355X peaks, and the per-class summary of a kernel trace,
on small hand-made rocprofv3-style files."""
import json
import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
import synth  # noqa: E402


def test_short_name_strips_namespace_and_arguments():
    n = "void (anonymous namespace)::k_conv_tile3<4, 8, false>(int const*, long, float const*)"
    assert bench._short_name(n) == "k_conv_tile3<4, 8, false>"
    assert bench._short_name("k_sum_split(float const*, int)") == "k_sum_split"
    # template arguments that hold parentheses stay whole
    assert bench._short_name("k_x<(anonymous namespace)::T(1)>(int)") == "k_x<T(1)>"


def test_op_rate_units_and_peaks():
    r = bench.op_rate("conv_fwd", 2e9, 1000.0, False)  # 2 GFLOP in 1 ms
    assert r["unit"] == "TFLOP/s" and r["achieved"] == pytest.approx(2.0)
    assert r["frac"] == pytest.approx(2.0 / 157.3, abs=1e-4)  # rounded to 4 places
    r = bench.op_rate("conv", 2e9, 1000.0, True)
    assert r["peak"] == 2500.0
    r = bench.op_rate("pool_fwd", 8e6, 10.0, False)  # 8 MB in 10 us
    assert r["unit"] == "GB/s" and r["achieved"] == pytest.approx(800.0)
    assert r["frac"] == pytest.approx(0.1)


def test_trace_classes():
    assert bench.trace_class("k_quant") == "build"
    assert bench.trace_class("k_leaf_mean") == "build"
    assert bench.trace_class("k_route_down<4>") == "pool"
    assert bench.trace_class("k_conv_dwt<false, 16, 2, 4, true, 2>") == "conv_main"
    assert bench.trace_class("k_cin_fwd<3, true>") == "conv_main"
    assert bench.trace_class("k_conv_tile3<2, 8, false, true>") == "conv_main"
    assert bench.trace_class("k_sum_parts<16, 4>") == "conv_helper"
    assert bench.trace_class("k_sum_split_pool") == "conv_helper"
    assert bench.trace_class("k_sr_table") == "conv_helper"
    assert bench.trace_class("at::native::vectorized_elementwise_kernel") == "other"


def _sizes(wl):
    """Small made-up per-depth sizes: N[l] = 8 M[l-1]."""
    M = [wl.batch * 2 ** l for l in range(wl.depth + 1)]
    N = [wl.batch] + [8 * M[l - 1] for l in range(1, wl.depth + 1)]
    return N, M


def test_conv_flops_by_hand():
    wl = synth.WORKLOADS["net_d5"]
    N, M = _sizes(wl)
    acc = bench.Accounting(wl, N, M, 1000)
    f, o = acc.conv_flops()
    want = 0
    for li, L in enumerate(wl.layers):
        if L.op == "conv":
            passes = 3 if li > 0 else 2  # the first layer has no input gradient
            want += passes * 2 * N[L.depth] * 27 * L.cin * L.cout
    assert f == want
    assert o == sum(N[L.depth] for L in wl.layers if L.op == "conv")


def test_summarize_trace(tmp_path, capsys):
    wl = synth.WORKLOADS["net_d5"]
    N, M = _sizes(wl)
    acc = bench.Accounting(wl, N, M, 1000)
    flops, _ = acc.conv_flops()
    line = {"metric": "m", "steps": 3, "warmup": 2, "ms_per_step": 1.0,
            "config": {"workload": "net_d5", "octants_per_depth": N, "nonempty_per_depth": M,
                       "points": 1000}}
    (tmp_path / "run.log").write_text("[bench] noise\n" + json.dumps(line) + "\n")
    d = tmp_path / "prof"
    d.mkdir()
    # 5 network steps (warmup 2 + 3 timed), 6 builds; times in ns
    rows = [("void (anonymous namespace)::k_conv_tile3<4, 8, false>(int)", 15, 15 * 40000),
            ("k_sum_split(float const*)", 10, 10 * 5000),
            ("k_pool_fwd<4>(float const*)", 20, 20 * 4000),
            ("k_quant(float const*)", 6, 6 * 7000),
            ("k_emit(int)", 6, 6 * 10000),
            ("at::native::copy(int)", 5, 5 * 2000)]
    with open(d / "run_kernel_stats.csv", "w") as fh:
        fh.write('"Name","Calls","TotalDurationNs","AverageNs","Percentage","MinNs","MaxNs","StdDev"\n')
        for name, calls, tot in rows:
            fh.write(f'"{name}",{calls},{tot},{tot / calls},1.0,{tot / calls},{tot / calls},0\n')
    bench.summarize_trace(str(d), str(tmp_path / "run.log"))
    out = capsys.readouterr().out
    # per step: conv main 15 * 40 / 5 = 120 us, helpers 10 * 5 / 5 = 10 us;
    # build (7 + 10) us per build; pooling 20 * 4 / 5 = 16 us
    assert "| conv fwd + bwd, main kernels | 120.0 |" in out
    assert "| conv fwd + bwd, every kernel | 130.0 |" in out
    assert "| build | 17.0 |" in out
    assert "| pool + unpool, fwd + bwd | 16.0 |" in out
    tf = flops / 120e-6 / 1e12
    assert f"{tf:.1f} TFLOP/s" in out
    assert "other kernels (at::native::copy)" in out
    assert "`k_conv_tile3<4, 8, false>` | 15 | 40.00 |" in out


def test_accounting_of_pool_backward():
    """The routing's bytes: per non-empty parent its gradient row, switches
    and row index, plus the pooled output when a ReLU'd convolution lies
    below (the ReLU's mask); every child row written."""
    N = [2, 16, 128, 1024]
    M = [2, 16, 100, 500]
    wl = synth.Workload("t", 0, 3, 2, 1000, "union", (
        synth.Layer("conv", 3, 3, 16, relu=True),
        synth.Layer("pool", 3, 16, 16),
        synth.Layer("conv", 2, 16, 16),
        synth.Layer("pool", 2, 16, 16),
    ), signal_input=False)
    acc = bench.Accounting(wl, N, M, 2000)
    _, p3, _, p2 = wl.layers
    assert acc.work("pool_bwd", p3) == M[2] * 16 * 9 + M[2] * 4 + N[3] * 16 * 4
    assert acc.work("pool_bwd", p2) == M[1] * 16 * 5 + M[1] * 4 + N[2] * 16 * 4


def test_accounting_of_deconvolution_gpool_and_stride4():
    """Flops and bytes of the ops added beside the convolution, computed by
    hand from the per-depth sizes."""
    N = [2, 16, 128, 1024, 8192]
    M = [2, 16, 100, 700, 3000]
    wl = synth.Workload("t", 0, 4, 2, 1000, "union", (
        synth.Layer("conv", 4, 3, 16),
        synth.Layer("conv", 4, 16, 32, stride=4),
        synth.Layer("deconv", 4, 32, 8, stride=2),
        synth.Layer("gpool", 4, 8, 8, ksize=5, mode="avg"),
        synth.Layer("gpool", 4, 8, 8, ksize=3, mode="max"),
    ), signal_input=False)
    acc = bench.Accounting(wl, N, M, 2000)
    c0, s4, dc, ga, gm = wl.layers
    # stride 4 from depth 4 is evaluated at the M[2] non-empty depth-2 octants
    # only; the stride-2 deconvolution to depth 4 runs the stride-2
    # convolution at depth 4 (evaluated at the M[3] non-empty depth-3 octants)
    assert acc.work("conv_fwd", s4) == 2 * M[2] * 27 * 16 * 32
    assert acc.work("deconv_fwd", dc) == 2 * M[3] * 27 * 32 * 8
    assert acc.work("deconv_bwd_weight", dc) == acc.work("deconv_fwd", dc)
    flops, octs = acc.conv_flops()
    assert flops == (4 * N[4] * 27 * 3 * 16 + 6 * M[2] * 27 * 16 * 32 + 6 * M[3] * 27 * 32 * 8)
    # output rows written: all depth-2 rows (stride 4), all depth-4 rows
    assert octs == N[4] + N[2] + N[4]
    # general pooling: rows in and out, switches for max, the groups' 27 entries
    assert acc.work("gpool_fwd", ga) == N[4] * 8 * 8 + M[3] * 108
    assert acc.work("gpool_bwd", gm) == N[4] * 8 * 8 + N[4] * 8 + M[3] * 108
    assert bench.BOUND["gpool_fwd"] == "hbm" and bench.BOUND["deconv_fwd"] == "mfma"
    assert bench.trace_class("k_gpool_fwd<2, true, 4>") == "pool"
    assert bench.trace_class("k_sr_mm<float, 0, 2, 2, 2, 2>") == "conv_main"
    assert bench.trace_class("k_sr_dw<unsigned short, 2, 2, 2, 1>") == "conv_main"
    assert bench.trace_class("k_sr_dyg<float>") == "conv_helper"
    assert bench.op_rate("deconv_fwd", 2e9, 1000.0, False)["unit"] == "TFLOP/s"
