"""bench.py end to end on the fp32 workload (256-wide layer, 2,048-token cache): the
JSON line, and the layer patch written by --dump-dw against the fp64 oracle (the
1e-4 bar for fp32 inputs)."""
import json
import os
import subprocess
import sys

import numpy as np
import pytest

import oracle
from workloads import CONFIGS, make_layer_inputs

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
pytestmark = pytest.mark.gpu


def test_bench_line_and_patch_dump(tmp_path):
    print("bench.py --config 0 --dump-dw", flush=True)
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--config", "0", "--steps",
                        "1", "--warmup", "0", "--no-cpu-baseline", "--dump-dw", str(tmp_path)],
                       capture_output=True, text=True, timeout=240, cwd=ROOT)
    assert r.returncode == 0, r.stderr[-2000:]
    line = json.loads(r.stdout.strip().splitlines()[-1])
    assert line["n_gpus"] == 1 and line["steps"] == 1 and line["value"] > 0
    assert line["roofline"]["frac"] > 0 and line["solve_info_nonzero_layers"] == 0
    dW = np.load(tmp_path / "dW_layer00.npy")
    cfg = CONFIGS[0]
    assert dW.shape == (cfg.d, cfg.d) and dW.dtype == np.float32
    ref = oracle.layer_patch(make_layer_inputs(cfg, 0), keep=False)["dW"]
    err = np.linalg.norm(dW - ref) / np.linalg.norm(ref)
    print(f"  dW vs oracle {err:.3e}", flush=True)
    assert err <= 1e-4
