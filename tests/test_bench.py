"""bench.py host logic (CPU): which bench lines may carry the counter-measured
HBM traffic of the committed rocprofv3 summary."""
import bench
import workloads as W

GU = "k_gemm_bf16_lds<2,8,64,1,0>"


def test_traffic_only_for_the_profiled_workload():
    for name in ("qwen3b_shape", "long_ragged_1p5b", "pool_3b", "tiny_f32"):
        assert bench.measured_traffic(GU, W.get_config(name)) is None, name
    c = W.get_config(bench.TRAFFIC_WORKLOAD)
    assert bench.measured_traffic(GU, W.fixed_k_variant(c), "fixed_k") is None
    assert bench.measured_traffic(GU, c, "sara", 0.9) is None
    assert bench.measured_traffic("no_such_kernel", c) is None


def test_profiled_traffic_is_consistent():
    c = W.get_config(bench.TRAFFIC_WORKLOAD)
    tr = bench.measured_traffic(GU, c)
    if tr is not None:   # the summary was taken on the current kernel source
        assert abs(tr["traffic"] / tr["alg_bytes_per_launch"] - tr["ratio"]) < 0.01
        assert tr["source"].startswith("profiles/")
