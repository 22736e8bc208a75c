"""CPU checks of bench.py's measurement arithmetic: the algorithmic FLOPs and bytes it divides by
come from the geometry formulas in bench.step_work / step_bytes; here they are recounted from the
weight tensor shapes (synth.tensor_specs) and the attention definition, for every workload. Also:
bench.py refuses more than one GPU with a message and exit status 2."""
import os
import subprocess
import sys

import numpy as np
import pytest

import bench
import synth

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _numel(specs, name):
    return int(np.prod([s for n, s, _ in specs if n == name][0]))


@pytest.mark.parametrize("key", ["c1", "c2", "c3", "c4", "c5"])
def test_flops_and_bytes_match_the_weight_shapes(key):
    w = synth.WORKLOADS[key]
    g = w.geom
    specs = synth.tensor_specs(g)
    T = w.batch * w.seq
    R = 123
    n = lambda name: _numel(specs, "l0." + name)
    layer_gemm = 2 * T * (n("wq") + n("wk") + n("wv") + n("wo") + n("wg") + n("wu") + n("wd"))
    # scores q.k and the P.V product: 2 * dh FLOPs each, per (query, key, head)
    attn = 2 * 2 * w.batch * g.n_heads * w.seq * (w.kv_prefix + w.seq) * g.head_dim
    lm = 2 * R * _numel(specs, "lm_head")
    assert bench.step_flops(w, R) == pytest.approx(g.n_layers * (layer_gemm + attn) + lm, rel=1e-12)
    by = bench.step_bytes(w, R)
    d, F = g.d_model, g.d_ffn
    assert by["gemm_gate_up_swiglu"] == 2 * (n("wg") + n("wu")) + 2 * T * d + 2 * T * F
    assert by["gemm_qkv_rope"] == 2 * (n("wq") + n("wk") + n("wv")) + 2 * T * d + 2 * T * (n("wq") + n("wk") + n("wv")) // d
    assert by["gemm_lm_head_top2"] == 2 * _numel(specs, "lm_head") + 2 * R * d


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True, text=True,
                       timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def test_stored_traffic_follows_the_kernel_source_digest(monkeypatch):
    """The committed counter traffic is reported only while the GEMM sources it was measured on are
    unchanged: a different digest drops it (the roofline then reports traffic as null)."""
    rec = bench.stored_traffic("gemm_gate_up_swiglu", "c2")
    if rec is not None:
        assert rec["source_digest"] == bench.kernel_source_digest()
        assert rec["hbm_bytes_per_launch"] == rec["fetch_bytes_per_launch"] + rec["write_bytes_per_launch"]
        assert rec["algorithmic_bytes_per_launch"] == \
            bench.step_bytes(synth.WORKLOADS["c2"], 256)["gemm_gate_up_swiglu"]
    monkeypatch.setattr(bench, "kernel_source_digest", lambda: "0" * 16)
    assert bench.stored_traffic("gemm_gate_up_swiglu", "c2") is None
    assert bench.stored_traffic("no_such_class", "c2") is None
