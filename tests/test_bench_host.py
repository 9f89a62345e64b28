"""bench.py's host-side contract and accounting, on the CPU (no GPU is touched).

The method's bytes and flops that bench.py prices its rooflines on are pinned to the figures the
layer's definition gives by hand at decode-20M (eq. (1): value rows of the bag, the selection and
the pooled output; eq. (2): the keys and queries of both axes), and the library's dispatch rules
that bench.py mirrors are checked against their stated conditions.
"""
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402
from synth import configs as CF  # noqa: E402


def test_more_than_one_gpu_exits_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr
    assert r.stdout == ""


def test_decode_method_bytes_by_hand():
    c = CF.C3
    assert (c.T, c.heads, c.n_keys, c.dk, c.topm, c.dv) == (32, 2, 4480, 128, 32, 512)
    w = bench.kernel_work(c, c.T, fused=True)
    keys = 2 * 2 * 4480 * 128 * 4                  # two axes, two heads, fp32 rows of 128
    queries = 2 * 32 * 2 * 128 * 4
    rows = 32 * 2 * 32 * 1024                      # 64 bf16 rows of 1 KiB per token
    sel_out = 32 * 2 * 32 * 8                      # idx and w
    pooled = 32 * 512 * 4
    assert w["axis_scores_kernel"]["bytes"] == keys + queries == 9_240_576
    assert w["select_kernel"]["bytes"] == rows + sel_out + pooled == 2_179_072
    assert w["select_kernel"]["intermediate"] == 2 * 32 * 2 * 4480 * 4 == 2_293_760
    assert w["axis_scores_kernel"]["bytes"] + w["select_kernel"]["bytes"] == 11_419_648
    assert w["axis_scores_kernel"]["flops"] == 4 * 32 * 2 * 4480 * 128


def test_layer_rules():
    # (project, fused): the selection pools only without projection or expansion, at most two
    # heads, m <= 64, rows of 1 or 2 KiB and T <= 128
    assert bench.layer_rules(CF.C3) == (False, True)
    assert bench.layer_rules(CF.C2) == (False, False)          # 2048 tokens
    assert bench.layer_rules(CF.C2.with_tokens(128)) == (False, True)
    assert bench.layer_rules(CF.C2.with_tokens(129)) == (False, False)
    assert bench.layer_rules(CF.C5) == (True, False)
    assert bench.layer_rules(CF.C6) == (True, False)


@pytest.mark.parametrize("name,T,want", [
    ("decode-20M", 32, False), ("decode-20M", 64, False), ("decode-20M", 65, True),
    ("prefill-1M", 2048, True), ("tucker-ive-4M", 4096, True), ("ultramem-1.6B-x12", 512, True),
])
def test_plane_scoring_rule(name, T, want):
    assert bench.scores_on_planes(CF.CONFIGS[name], T) is want


def test_scoring_roofline_priced_on_its_mfma_type():
    # many tokens on the fp16 planes: the method's flops against the fp16 peak, the issued fp16
    # work (three products per method flop) and the fp32 fraction beside
    c = CF.C2
    flops = 4 * c.T * c.heads * c.n_keys * c.dk
    r = bench.roofline_for(c, c.T, "axis_scores_kernel", 20.0, "not-profiled", False)
    assert r["bound"] == "mfma" and r["peak"] == bench.F16_PEAK_TFLOPS
    assert r["achieved"] == pytest.approx(flops / 20e-6 / 1e12, rel=1e-3)
    assert r["issued_fp16_TFLOPs"] == pytest.approx(3 * r["achieved"], rel=1e-3)
    assert r["frac_of_fp32_peak"] == pytest.approx(r["achieved"] / bench.FP32_PEAK_TFLOPS, rel=1e-3)
    assert r["traffic"] is None
    # decode: the keys dominate, HBM-bound
    d = CF.C3
    r = bench.roofline_for(d, d.T, "axis_scores_kernel", 5.0, "not-profiled", True)
    assert r["bound"] == "hbm" and r["peak"] == bench.HBM_PEAK_GBS
    assert r["algorithmic_bytes"] == 9_240_576


def test_decode_select_roofline_bytes():
    c = CF.C3
    r = bench.roofline_for(c, c.T, "select_kernel", 10.0, "not-profiled", True)
    assert r["bound"] == "hbm"
    assert r["algorithmic_bytes"] == 2_179_072
    assert r["achieved"] == pytest.approx(2_179_072 / 10e-6 / 1e9, rel=1e-3)
    assert r["intermediate_bytes"] == 2_293_760


def test_warm_replays_until_the_time_has_passed():
    # the untimed warm-up before each timed region: at least one replay, and replays (each
    # followed by a device synchronisation) until the given wall time has passed
    import time as _time

    class _Cuda:
        syncs = 0

        @classmethod
        def synchronize(cls):
            cls.syncs += 1

    class _Torch:
        cuda = _Cuda

    calls = []
    bench.warm(lambda: calls.append(1), _Torch, 0.0)
    assert len(calls) == 1 and _Cuda.syncs == 1
    t0 = _time.perf_counter()
    bench.warm(lambda: (calls.append(1), _time.sleep(0.002)), _Torch, 0.02)
    assert _time.perf_counter() - t0 >= 0.02
    assert len(calls) >= 1 + 5 and _Cuda.syncs == len(calls)
