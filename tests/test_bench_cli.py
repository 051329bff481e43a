"""bench.py's host-side contract, on the CPU: the one-GPU refusal, the traffic table's validity
check, and the workload names (no GPU, no library call)."""
import os
import subprocess
import sys

import bench
from paper_2606_26453_amd import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, "bench.py", "--gpus", "2"], cwd=ROOT, capture_output=True, text=True,
                       timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_code_hash_ignores_comments_and_blank_lines():
    a = "int x = 1;  // one\n\n  return x;\n"
    b = "int x = 1;\n  return x;   // two\n"
    assert bench.code_hash(a) == bench.code_hash(b)
    assert bench.code_hash(a) != bench.code_hash(a.replace("1", "2"))


def test_traffic_is_reported_only_for_the_measured_code(monkeypatch):
    for call, (group, f, w) in bench.TRAFFIC_KIB.items():
        files = bench.TRAFFIC_SOURCES[group][0]
        src = {g: (fs, bench.source_hash(fs)) for g, (fs, _) in bench.TRAFFIC_SOURCES.items()}
        monkeypatch.setattr(bench, "TRAFFIC_SOURCES", src)
        assert bench.measured_traffic(call, bench.TRAFFIC_CONFIG) == int(f * bench.FETCH_SCALE + w * bench.WRITE_SCALE)
        assert bench.measured_traffic(call, bench.TRAFFIC_CONFIG + 1) is None   # another workload
        monkeypatch.setattr(bench, "TRAFFIC_SOURCES", dict(src, **{group: (files, "0" * 16)}))
        assert bench.measured_traffic(call, bench.TRAFFIC_CONFIG) is None        # the kernels changed since
        monkeypatch.setattr(bench, "TRAFFIC_SOURCES", src)
        assert bench.measured_traffic(call, bench.TRAFFIC_CONFIG, variant=True) is None   # other kernels
    assert bench.measured_traffic("no_such_call", bench.TRAFFIC_CONFIG) is None


def test_measured_traffic_covers_every_layer_call():
    # every call of the default layer step has counter bytes, and none moves fewer bytes than it
    # must (the unique bytes of the HBM-bound calls; the MFMA calls' operands and outputs)
    from paper_2606_26453_amd.layer import MoELayer
    lay = object.__new__(MoELayer)
    lay.cfg, lay.fp8, lay.gather_fused, lay.shared = W.CONFIGS[bench.TRAFFIC_CONFIG], False, False, False
    lay.router_fused_dx = False
    lay.fp8_bwd = lay.mx = lay.fp8_dw = False
    work = lay.work()
    c = lay.cfg
    R = c.T * c.k
    operands = {"fwd_gate_up": R * c.d * 2 + 2 * c.E * c.d * c.f * 2 + 3 * R * c.f * 2,
                "fwd_down": R * c.f * 2 + c.E * c.f * c.d * 2 + R * c.d * 2,
                "dw_down": R * c.f * 2 + R * c.d * 2 + c.E * c.f * c.d * 4,
                "dx_down_swiglu_bwd": R * c.d * 2 + c.E * c.f * c.d * 2 + 4 * R * c.f * 2,
                "dx_gate_up": 2 * R * c.f * 2 + 2 * c.E * c.d * c.f * 2 + R * c.d * 2,
                "dw_gate_up": R * c.d * 2 + 2 * R * c.f * 2 + 2 * c.E * c.d * c.f * 4}
    step_calls = {"route_permute", "fwd_gate_up", "fwd_down", "combine", "combine_bwd", "dw_down",
                  "dx_down_swiglu_bwd", "dx_gate_up", "unpermute_dx", "dw_gate_up"}
    assert set(bench.TRAFFIC_KIB) == step_calls
    for call, (_, f, w) in bench.TRAFFIC_KIB.items():
        hbm = f * bench.FETCH_SCALE + w * bench.WRITE_SCALE
        need = work[call][1] if work[call][0] == "bytes" else operands[call]
        assert hbm >= 0.999 * need, call


def test_workload_names():
    assert bench.workload_name(1, W.CONFIGS[1]) == "config 1: mixtral MoE FFN layer fwd+bwd"
    assert bench.workload_name(1, W.CONFIGS[1], router=True).endswith("incl. router")
    n5 = bench.workload_name(5, W.CONFIGS[5])
    assert "dW1" in n5 and "bf16 output" in n5 and "alpha=0.24" in n5
    assert "fp32 output" in bench.workload_name(4, W.CONFIGS[4])


def test_step_statistics():
    st = bench._stats([5.0, 1.0, 3.0, 2.0, 4.0, 6.0, 7.0, 8.0, 9.0, 10.0, 11.0])
    assert st["median"] == 6.0 and st["p10"] == 2.0 and st["p90"] == 10.0
    assert st["min"] == 1.0 and st["max"] == 11.0


def test_vector_alu_calls_are_scored_against_their_roof():
    # the router's logits at the Mixtral shape: 2*T*d*E FLOP over ~2*T*d bytes -> E FLOP/B = 8,
    # below the 19.7 FLOP/B ridge: HBM-bound, scored against 8 TB/s
    T, d, E = 8192, 4096, 8
    r = bench.valu_record(2 * T * d * E, T * d * 2 + d * E * 4 + T * E * 4, 0.05)
    assert r["bound"] == "hbm" and abs(r["frac_peak"] - r["gbs"] / 8000.0) < 1e-3
    assert abs(bench.VALU_RIDGE - 19.6625) < 1e-3
    # 64 FLOP/B: above the ridge, scored against the fp32 vector peak
    r = bench.valu_record(64e9, 1e9, 1.0)
    assert r["bound"] == "valu" and abs(r["frac_peak"] - 64.0 / 157.3) < 1e-3
