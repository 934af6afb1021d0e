"""Host-side logic of bench.py (CPU): the overlap and prediction metrics, the
committed traffic summary it reads, and the one-GPU guard."""
import os
import subprocess
import sys

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
sys.path.insert(0, ROOT)

import bench  # noqa: E402


def _stats(high, low=0, stall_ms=0.0, **kw):
    s = {"bytes_high": high, "bytes_low": low, "stall_ms": stall_ms}
    s.update(kw)
    return s


def test_overlap_closed_form():
    # 10 GB at 50 GB/s = 0.2 s of load; 0.05 s stalled over a 1 s run
    m = bench.overlap_metrics(_stats(10e9, stall_ms=50.0), 1.0, 50.0)
    assert m["load_s"] == pytest.approx(0.2)
    assert m["H_time"] == pytest.approx(0.75)
    assert m["H_max"] == pytest.approx(1.0)  # (1 - 0.05) / 0.2 > 1: capped


def test_overlap_never_prices_the_link_below_the_run():
    # the run moved 54 GB/s while the probe read 52: the load uses 54, so the
    # load cannot exceed the elapsed time and H_time cannot exceed H_max
    s = _stats(54e9, stall_ms=800.0)
    m = bench.overlap_metrics(s, 1.0, 52.0)
    assert m["load_s"] == pytest.approx(1.0)
    assert m["H_max"] <= 1.0
    assert m["H_time"] <= m["H_max"] + 1e-12


def test_overlap_without_copies():
    assert bench.overlap_metrics(_stats(0), 1.0, 50.0) is None


def test_prediction_metrics():
    s = {"pred_n": 100, "pred_correct": 70, "pred_in_time": 35, "spec_used": 20, "miss": 30}
    m = bench.prediction_metrics(s)
    assert m["accuracy"] == pytest.approx(0.7)
    assert m["fetch_rate"] == pytest.approx(0.5)
    assert m["goodpred"] == pytest.approx(0.35)
    assert m["proactive_coverage"] == pytest.approx(0.4)
    assert bench.prediction_metrics({"pred_n": 0, "pred_correct": 0, "pred_in_time": 0, "spec_used": 0,
                                     "miss": 0})["accuracy"] is None


def test_traffic_summary_is_tied_to_the_kernel_source():
    # the summary's figures are used only while the GEMV source (and the device
    # helpers it inlines) still hashes to the digest recorded with them; a
    # changed kernel reports no traffic
    import hashlib
    csrc = os.path.join(ROOT, "paper_2410_22134_amd", "csrc")
    src = b"".join(open(os.path.join(csrc, f), "rb").read() for f in ("kernels_gemv.hip", "common.hpp"))
    digest = hashlib.sha256(src).hexdigest()[:16]
    line = [l.split() for l in open(os.path.join(ROOT, "profiles", "traffic_counters.txt"))
            if l.startswith("traffic k_ffn_gateup")][0]
    traffic, ratio = bench.read_traffic("k_ffn_gateup")
    if line[2] == digest:
        assert traffic == int(line[3])
        assert ratio == pytest.approx(int(line[3]) / int(line[4]), abs=1e-4)  # bench rounds to 4 places
    else:
        assert (traffic, ratio) == (None, None)
    assert bench.read_traffic("no_such_kernel") == (None, None)


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=300, cwd=ROOT)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


class _HostModel:
    """The host views bench's oracle timing reads (weights as data), built from the
    seeded recipes without a GPU."""

    def __init__(self, cfg):
        import numpy as np
        from synth import model as sm
        self.cfg = cfg
        self.np_gate = [sm.gate(cfg, l) for l in range(cfg.n_layers)]
        self.np_bias = [sm.bias(cfg, l) for l in range(cfg.n_layers)]
        self.np_pred = [sm.predictor(cfg, l) for l in range(cfg.n_layers)]
        self.np_sgate = [sm.shared_gate_vec(cfg, l) for l in range(cfg.n_layers)]
        self._buf = {}
        for l in range(cfg.n_layers):
            for e in range(cfg.n_experts):
                b = np.zeros(cfg.expert_bytes, np.uint8)
                sm.write_expert(cfg, l, e, b.ctypes.data)
                self._buf[l, e] = b

    def expert_host(self, l, e):
        import numpy as np
        b = self._buf[l, e]
        if self.cfg.weight_format == "int4":
            return b
        return b.view(np.uint16 if self.cfg.dtype == "bf16" else np.float32)


@pytest.mark.parametrize("fmt,T", [("dense", 1), ("dense", 7), ("int4", 3)])
def test_oracle_rate_on_a_small_model(fmt, T):
    sys.path.insert(0, HERE)
    import parity_util as pu
    cfg = pu.SMALL.with_(weight_format=fmt)
    r = bench.oracle_rate(cfg, _HostModel(cfg), T, 0.05)
    assert r["value"] > 0 and r["kind"] == "oracle" and r["unit"] == "tok/s" and r["cores"] >= 1


def test_summary_line_reads_every_leg():
    k = {"gemv_gateup": {"frac_hbm": 0.7}, "gemv_down": {"frac_hbm": 0.6}}
    out = {"value": 37.0, "roofline": {"frac": 0.6, "down": {"frac": 0.5}},
           "detail": {"overlap": {"H_time_over_H_max": 0.8}, "prediction": {"goodpred": 0.35, "accuracy": 0.7},
                      "allres": {"tok_s": 500.0, "of_ceiling": 0.25, "kernels": k},
                      "prefill": {"tok_s": 2100.0},
                      "configs": {"Mixtral-8x7B int4": {"runs": [{"workload": "prefill", "tokens_per_step": 256,
                                                                  "tok_s": 900.0},
                                                                 {"workload": "decode", "tokens_per_step": 1,
                                                                  "tok_s": 14.0}]}},
                      "predictor_training": {"lookahead_1": {"heldout_acc_trained": {"mean": 0.73}},
                                             "lookahead_2": {"heldout_acc_trained": {"mean": 0.71}}}},
           "roofline_prefill_gemm": {"frac": 0.44}, "cpu_baseline": {"value": 0.26}}
    line = bench.summary_line(out)
    for piece in ("decode 37.0 tok/s", "all-resident 500.0", "Mixtral-8x7B int4: prefill 900.0, decode b1 14.0",
                  "shared GEMM 0.440", "GoodPred 0.350", "oracle 0.26"):
        assert piece in line, (piece, line)


def test_traffic_is_scaled_to_the_run():
    # the counter runs' bytes-over-algorithmic ratio, applied to this run's launches
    assert bench.traffic_here(1.01, {"bytes_per_launch": 1000}) == 1010
    assert bench.traffic_here(None, {"bytes_per_launch": 1000}) is None
    assert bench.traffic_here(1.01, {}) is None
