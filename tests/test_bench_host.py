"""Host-side pieces of bench.py: the kernel-source hash that decides whether a
committed traffic measurement still applies, and the --gpus contract."""
import os
import subprocess
import sys

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_code_only_drops_comments_not_literals():
    src = ('int a = 1; // trailing\n'
           'const char* s = "x // kept /* kept */"; /* block\n spanning */ int b = \'/\';\n'
           'char q = \'"\'; // after a quote character\n')
    got = " ".join(bench._code_only(src).split())
    assert got == 'int a = 1; const char* s = "x // kept /* kept */"; int b = \'/\'; char q = \'"\';'


def test_source_hash_ignores_comments_and_layout(tmp_path, monkeypatch):
    csrc = tmp_path / "paper_2604_21290_amd" / "csrc"
    csrc.mkdir(parents=True)
    (csrc / "k.hip").write_text("__global__ void k(int* p) { p[0] = 1; }\n")
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    h0 = bench.kernel_source_sha()
    (csrc / "k.hip").write_text("// what k does\n__global__ void k(int* p) {\n  p[0] = 1;  /* one */\n}\n")
    assert bench.kernel_source_sha() == h0
    (csrc / "k.hip").write_text("__global__ void k(int* p) { p[0] = 2; }\n")
    assert bench.kernel_source_sha() != h0


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode != 0
    assert "one GPU" in (r.stdout + r.stderr) or "1 GPU" in (r.stdout + r.stderr)


def test_cpu_baseline_runs_the_oracle_in_worker_processes():
    from paper_2604_21290_amd import inputs as I
    w = I.WORKLOADS["single"]
    r = bench.cpu_baseline(w, images=1, min_seconds=0.2)
    assert r["kind"] == "oracle" and r["unit"] == "layers/s"
    assert r["value"] > 0 and r["cores"] == 1
    assert "single-thread processes" in r["sample"]


def test_layer_work_matches_the_per_config_table():
    """One layer's algorithmic flop and bytes (one build + one update) for the
    five configurations: Gram 2BNMC + FC 4BNC^2 flop; bytes counted once each
    (X by the build and by the update, pooled keys, the graph written and
    read, W, the output, the pooling's own I/O)."""
    from paper_2604_21290_amd import inputs as I
    want = {  # name: (GFLOP, MB) as the per-config table prints them (3 digits)
        "single": (0.044, 0.76), "vig_ti": (1.40, 7.8), "vig_b": (23.7, 50.7),
        "pyr_s1": (5.72, 74.5), "pyr_s2": (4.14, 40.0), "hires": (16.0, 17.7),
    }
    for name, (gf, mb) in want.items():
        w = I.WORKLOADS[name]
        F, Y = bench.layer_work(w, 2 if w.dtype == I.BF16 else 4)
        assert abs(F / 1e9 - gf) / gf < 1e-2, (name, F)
        assert abs(Y / 1e6 - mb) / mb < 1e-2, (name, Y)
    assert bench.layer_work(I.WORKLOADS["vig_ti"], 2)[1] == 7824384
