"""bench.py's headline record on the CPU: the compulsory bytes and the method's
flops of the headline workload against their closed forms (Q, K, V read and
O written once, 4 N d s bytes per head; 2 x the MACs T (2 N b d + 2 N m d) +
N b d per head, the work count that reproduces the paper's attention-FLOP
tables), the call roofline built from them, and a record with every field at
its widest that still fits the 4 KB a log tail keeps whole."""
import importlib.util
import json
import os

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


@pytest.fixture(scope="module")
def bench():
    spec = importlib.util.spec_from_file_location("bench_under_test", os.path.join(ROOT, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


@pytest.fixture(scope="module")
def headline():
    import synth_inputs as si

    return si.WORKLOADS["speed_n16384"]


def test_headline_work(bench, headline):
    w = headline
    assert (w.B, w.H, w.N, w.m, w.b, w.d, w.T, w.dtype) == (1, 16, 16384, 128, 128, 64, 2, "bf16")
    nbytes, flops = bench.call_work(w)
    heads, n, m, b, d, T = w.B * w.H, w.N, w.m, w.b, w.d, w.T
    assert nbytes == heads * 4 * n * d * 2 == 134217728
    macs = T * (2 * n * b * d + 2 * n * m * d) + n * b * d
    assert flops == heads * 2 * macs == 38654705664


def test_call_roofline_is_compulsory_bytes_over_time(bench, headline):
    ms = 0.112  # a call of 112 us
    kernels = [{"kernel": k, "avg_us": us, "alg_bytes": 10**8, "alg_flops": 10**10}
               for k, us in (("r_half_step", 24.0), ("l_half_step", 26.0), ("r_half_step_final", 35.0),
                             ("monarch_apply", 27.0))]
    roof = bench.headline_roofline(headline, ms, kernels, {"copy_GB_s": 5000.0, "gemm_bf16_TFLOP_s": 1000.0})
    # HBM binds: 134 MB at 8 TB/s (16.8 us) against 38.7 GFLOP at 2.5 PFLOP/s (15.4 us)
    assert roof["bound"] == "hbm" and roof["unit"] == "GB/s" and roof["scope"] == "call"
    assert roof["achieved"] == pytest.approx(134217728 / 112e-6 / 1e9, abs=0.1)
    assert roof["frac"] == pytest.approx(134217728 / 112e-6 / 8e12, abs=1e-4)
    assert roof["frac_of_measured"] == pytest.approx(roof["achieved"] / 5000.0, abs=1e-4)
    assert roof["dominant_kernel"]["kernel"] == "r_half_step_final"
    assert roof["dominant_kernel"]["launches"] == 4


def test_record_fits_and_carries_the_contract(bench, headline):
    w = headline
    ms = 0.1234567891
    kernels = [{"kernel": k, "avg_us": 33.333333, "alg_bytes": 169869312, "alg_flops": 12884901888}
               for k in ("r_half_step", "l_half_step", "r_half_step_final", "monarch_apply")]
    roof = bench.headline_roofline(w, ms, kernels, {"copy_GB_s": 5076.7123, "gemm_bf16_TFLOP_s": 1076.0123})
    roof["traffic"] = 532162251123  # widest plausible figure
    cfg = {"workload": w.name, "B": w.B, "H": w.H, "N": w.N, "m": w.m, "b": w.b, "d": w.d, "T": w.T,
           "inputs": w.recipe, "alpha": 1.6676876659127036, "rotating_input_sets": 4}
    also = [{"workload": name, "value": 4452003625.912345, "ms_per_step": 0.016992123, "roofline_frac": 0.28491234,
             "bound": "hbm"} for name in ("speed_n4096", "vit_b16_n196", "speed_n4096_t3", "vit_b16_n197",
                                           "roberta_n1024")]
    value = w.B * w.H * w.N / (ms * 1e-3)
    rec = bench.compact_record(w, value, ms, 50, 10, cfg, roof, also)
    rec["cpu_baseline"] = {"value": 392175.812345, "unit": "heads*tokens/s", "cores": 128, "kind": "oracle",
                           "sample": "15 full forward passes of speed_n16384 (all 16 heads), fp64, 10.0s",
                           "single_thread": {"value": 383187.812345, "unit": "heads*tokens/s", "cores": 1,
                                             "sample": "20 passes of vit_b16_n196 at B=4 (48 heads), fp64, "
                                                       "1 thread, 0.5s"}}
    rec["details"] = "gpurun_out/bench_details_with_a_long_name.json"
    line = bench.record_line(rec)
    assert len(line) < 4096 and "\n" not in line
    back = json.loads(line)
    for key in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step", "higher_is_better",
                "scaling", "vs_baseline", "dtype", "data", "config", "roofline", "cpu_baseline"):
        assert key in back, key
    assert back["n_gpus"] == 1 and back["vs_baseline"] is None and back["higher_is_better"] is True
    assert back["config"]["workload"] == "speed_n16384"
    for key in ("bound", "achieved", "peak", "unit", "frac", "traffic"):
        assert key in back["roofline"], key
    for key in ("value", "unit", "cores", "kind", "sample"):
        assert key in back["cpu_baseline"], key
    assert back["value"] == pytest.approx(16 * 16384 / (ms * 1e-3), rel=1e-9)
