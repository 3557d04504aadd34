"""Host-side checks of bench.py: the one-GPU refusal, and the code hash that
keys the stored contraction traffic (it must ignore comments and whitespace
and see every change to the code)."""
import importlib.util
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _bench():
    spec = importlib.util.spec_from_file_location("bench_mod", os.path.join(ROOT, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


SRC = """// header comment
template <int N> __global__ void k(float* a) {  /* block
   comment */
    a[threadIdx.x] *= 2.f;   // trailing
}
"""


def test_code_hash_ignores_comments_and_whitespace(tmp_path):
    b = _bench()
    p0, p1, p2 = tmp_path / "a.hip", tmp_path / "b.hip", tmp_path / "c.hip"
    p0.write_text(SRC)
    p1.write_text(SRC.replace("// trailing", "// another remark")
                     .replace("block\n   comment", "x").replace("    a[", "\ta["))
    p2.write_text(SRC.replace("2.f", "3.f"))
    h0, h1, h2 = (b.kernel_code_hash(str(p)) for p in (p0, p1, p2))
    assert h0 == h1
    assert h0 != h2


def test_stored_traffic_is_keyed_by_the_code_hash():
    b = _bench()
    import json
    d = json.load(open(os.path.join(ROOT, "profiles", "igemm_vgg19_traffic.json")))
    assert "igemm_code_sha256_16" in d and d["bytes_per_step"] > 0
    # reported only while the stored hash matches the current kernel code
    expect = d["bytes_per_step"] if d["igemm_code_sha256_16"] == b.kernel_code_hash() else None
    assert b.measured_traffic("vgg19") == expect


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=300, cwd=ROOT)
    assert r.returncode != 0
    assert "one GPU" in (r.stdout + r.stderr)


def test_cpu_baseline_only_runs_the_oracle_without_a_gpu():
    import json
    env = dict(os.environ, OMP_NUM_THREADS="1")
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--cpu-baseline-only",
                        "--workload", "tiny", "--cpu-images", "2"],
                       capture_output=True, text=True, timeout=300, cwd=ROOT, env=env)
    assert r.returncode == 0, r.stderr[-2000:]
    d = json.loads(r.stdout.strip().splitlines()[-1])
    assert d["kind"] == "oracle" and d["cores"] == 1 and d["value"] > 0
    assert d["unit"] == "images/s" and "2 image(s)" in d["sample"]


def test_per_layer_work_sums_to_the_step_flop():
    # the per-layer forward and backward FLOP add up to the step's
    # contraction FLOP, for every workload's layer list
    b = _bench()
    sys.path.insert(0, ROOT)
    from paper_2005_14038_amd import workloads
    for name, wl in workloads.WORKLOADS.items():
        layers = wl.builder().layers
        rows = b.layer_work(layers, wl.batch, wl.H, wl.W, wl.C, need_dx=wl.need_dx)
        assert len(rows) == len(layers)
        total = sum(r["fwd_flop"] + r["bwd_flop"] for r in rows)
        assert total == b.contraction_flops(layers, wl.batch, wl.H, wl.W, wl.C,
                                            need_dx=wl.need_dx), name
        assert all(r["fwd_bytes"] > 0 and r["bwd_bytes"] > 0 for r in rows), name


def test_per_layer_rooflines_fractions():
    b = _bench()
    rows = [{"layer": 0, "op": "conv", "out": [1, 1, 8], "fwd_flop": 2e9, "bwd_flop": 4e9,
             "fwd_bytes": 1e6, "bwd_bytes": 2e6},
            {"layer": 1, "op": "relu", "out": [1, 1, 8], "fwd_flop": 0, "bwd_flop": 0,
             "fwd_bytes": 8e6, "bwd_bytes": 8e6}]
    out = b.per_layer_rooflines(rows, [0.2, 0.0], [0.4, 0.0], 10, 157.3)
    assert [e["pass"] for e in out] == ["fwd", "bwd"]      # the ReLU launched nothing
    e = out[0]
    assert abs(e["TFLOP/s"] - 2e9 / 0.02e-3 / 1e12) < 1e-6
    assert abs(e["attainable"] - 1.0) < 1e-9              # 2000 FLOP/B is above the ridge
    assert e["bound"] == "mfma"


def test_step_flop_of_the_five_workloads():
    """Contraction FLOP per minibatch step (2 per multiply-add; forward, data
    gradient and weight gradient; no data gradient for the layer reading the
    image; the ResNet-152 middle stage hands its input gradient back), from
    the per-image forward multiply-adds of the networks: 0.36 M, 11.18 G,
    19.63 G, 9.92 G, 11.51 G."""
    b = _bench()
    sys.path.insert(0, ROOT)
    from paper_2005_14038_amd import workloads
    want = {"tiny": 8.2e6, "vgg19_s1": 2.142e12, "vgg19": 3.764e12,
            "resnet152_mid": 1.904e12, "resnet152": 2.203e12}
    for name, wl in workloads.WORKLOADS.items():
        f = b.contraction_flops(wl.builder().layers, wl.batch, wl.H, wl.W, wl.C,
                                need_dx=wl.need_dx)
        assert abs(f / want[name] - 1) < 2e-3, (name, f)
    assert workloads.WORKLOADS["resnet152_mid"].need_dx
    assert not any(w.need_dx for n, w in workloads.WORKLOADS.items() if n != "resnet152_mid")
