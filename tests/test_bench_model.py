"""The bench line's roofline selection and algorithmic work model (CPU):
which roof each stage is priced against, the fp32 transform's peak (the
bf16 dense peak over its six part products), the ridge points, and the
work model's counts for the device<-op records and the message table."""
import math

import pytest

import bench
import synth


def _work(name, stage):
    wl = synth.WORKLOADS[name]
    topo = synth.make_topology(name)
    return wl, topo, bench.algorithmic_work(stage, wl, topo, wl.batch, None, wl.n_slices, 0)


def test_fp32_transform_peak_is_bf16_peak_over_six_part_products():
    assert bench.TRANSFORM_PEAK["f32"] == pytest.approx(2500.0 / 6)
    assert bench.TRANSFORM_PEAK["bf16"] == 2500.0


def test_transform_flops_are_the_fp32_contraction():
    wl, topo, (flops, _) = _work("transformer", "transform")
    rows = wl.batch * (topo.n_op + topo.n_dev)
    assert flops == pytest.approx(2.0 * rows * wl.f * 2 * wl.f)


@pytest.mark.parametrize("name,bound", [("transformer", "mfma"), ("sweep", "hbm"), ("large", "hbm"), ("cnn", "hbm")])
def test_transform_roof_follows_the_ridge(name, bound):
    # f = 256 fp32: 85 flop/B, above the split peak's 52 flop/B ridge; f = 128
    # fp32 (41 flop/B) and bf16 (171 < 312 flop/B) are HBM-bound
    wl, _, (flops, byts) = _work(name, "transform")
    ridge = bench.TRANSFORM_PEAK[wl.dtype] * 1e12 / (bench.PEAK_HBM_GBS * 1e9)
    assert (flops / byts >= ridge) == (bound == "mfma")
    avg_s = 1e-3
    roof = bench.nearest_roof("transform", wl.dtype, flops, byts, avg_s)
    assert roof["bound"] == bound
    if bound == "mfma":
        assert roof["peak"] == pytest.approx(416.67, abs=0.01)
        assert roof["frac"] == pytest.approx(flops / avg_s / 1e12 / (2500.0 / 6), abs=1e-4)
        assert "peak_basis" in roof
    else:
        assert roof["peak"] == bench.PEAK_HBM_GBS
        assert roof["achieved"] == pytest.approx(byts / avg_s / 1e9, abs=0.1)


def test_aggregation_roof_takes_the_nearer_of_valu_and_hbm():
    peak_valu = 256 * 4 * 16 * 2 * 2.4e9 / 1e12
    assert bench.PEAK_VALU_F32_TFLOPS == pytest.approx(peak_valu)
    # 40 TFLOP/s of vector work and 1 TB/s: the VALU fraction (0.51) is the larger
    roof = bench.nearest_roof("agg_op_dev", "bf16", 40e12 * 1e-3, 1e12 * 1e-3, 1e-3)
    assert roof["bound"] == "alu" and roof["frac"] == pytest.approx(40 / peak_valu, abs=1e-4)
    assert roof["hbm_frac"] == pytest.approx(1000 / bench.PEAK_HBM_GBS, abs=1e-4)
    # 5 TFLOP/s and 6 TB/s: HBM is the nearer roof
    roof = bench.nearest_roof("agg_dev_op", "f32", 5e12 * 1e-3, 6e12 * 1e-3, 1e-3)
    assert roof["bound"] == "hbm" and roof["frac"] == pytest.approx(0.75, abs=1e-4)


@pytest.mark.parametrize("name", ["cnn", "transformer", "large"])
def test_work_model_counts_records_and_table(name):
    wl, topo, (_, by_dev) = _work(name, "agg_dev_op")
    _, _, (_, by_merge) = _work(name, "agg_dev_merge")
    N, M, F, K, R = topo.n_op, topo.n_dev, wl.f, wl.heads, wl.batch
    tiles = -(-N // 64)
    groups = tiles if tiles <= 8 else -(-tiles // -(-tiles // 8))
    assert groups <= 8
    rec = R * M * groups * (F + 2 * K) * 4
    s = 2 if wl.dtype == "bf16" else 4
    assert by_dev == pytest.approx(R * N * F * s + R * N * 16 + R * N * 2 * K * 4 + R * M * K * 4 + rec)
    _, _, (_, by_prep) = _work(name, "dev_prep")
    t = R * M * F * (12 if (wl.dtype == "bf16" or F >= 256) else 8)
    assert by_prep == pytest.approx(R * (N + M) * 2 * F * s + t + R * (N + M) * 4 * K * 4)
    assert math.isfinite(by_merge) and by_merge > rec
