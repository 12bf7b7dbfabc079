"""bench.py's command-line contract, checked on a host without a GPU: it
refuses more than one GPU, and its JSON line carries every required field
(the line is built from a synthetic result here; no kernel runs)."""
import json
import os
import subprocess
import sys
import types

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_json_line_contract(capsys):
    sys.path.insert(0, ROOT)
    import bench
    from paper_2607_19547_amd import synth
    w = synth.WORKLOADS["long65k"]
    args = types.SimpleNamespace(steps=10, warmup=2, batched_layers=0)
    flops = 1.7e12
    r = dict(ms=60.0, steps=10, n_sel=6349, attn_flops_per_layer=flops, rebase_bytes=2340421632,
             trace={"sel_attn_mfma": (360, 10 * 36 * 1.6), "rebase_bf16_d128": (10, 10 * 0.4),
                    "scatter_rows": (360, 3.0), "sel_attn_combine": (360, 11.0)})
    rho1 = dict(ms=520.0)
    cpu = dict(value=4.4e5, unit="ms", cores=16, kind="oracle", sample="one layer, extrapolated")
    bench.emit(args, w, 0.1, r, rho1, cpu, gemm=dict(shape=[8192, 8192, 16384], ms=1.75, TFLOPs=1250.0))
    line = json.loads(capsys.readouterr().out.strip().splitlines()[-1])
    for key in ("metric", "value", "unit", "n_gpus", "steps", "warmup", "ms_per_step", "higher_is_better",
                "scaling", "vs_baseline", "dtype", "data", "config", "roofline", "cpu_baseline"):
        assert key in line, key
    assert line["n_gpus"] == 1 and line["higher_is_better"] is False and line["value"] == 60.0
    assert "workload" in line["config"] and "model" not in line["config"]
    roof = line["roofline"]
    assert roof["bound"] == "mfma" and roof["unit"] == "TFLOP/s" and roof["peak"] == 2500.0
    # achieved = algorithmic flop per launch / average launch duration
    assert roof["achieved"] == pytest.approx(flops / 1.6e-3 / 1e12, rel=1e-3)
    assert roof["frac"] == pytest.approx(roof["achieved"] / roof["peak"], rel=1e-3)
    assert "traffic" in roof
    assert line["roofline_rebase"]["bound"] == "hbm" and line["roofline_rebase"]["peak"] == 8000.0
    assert line["cpu_baseline"]["kind"] == "oracle" and line["cpu_baseline"]["cores"] == 16
    assert line["rho1_over_rho_speedup"] == pytest.approx(520.0 / 60.0, rel=1e-3)
    assert line["context_vendor_gemm_bf16"]["sel_attn_over_gemm"] == pytest.approx(roof["achieved"] / 1250.0,
                                                                                   rel=1e-3)
