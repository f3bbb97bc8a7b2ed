"""CPU checks of bench.py's host logic: the one-GPU guard, the workload
tables, the code digest that keys the committed HBM counters, the error
measure against the oracle, and the oracle baseline leg on a tiny call."""
from __future__ import annotations

import os
import shutil
import subprocess
import sys

import numpy as np

import bench
import oracle
from paper_2609_38981_amd import workloads as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_exits_with_a_message():
    r = subprocess.run([sys.executable, "bench.py", "--gpus", "2"], cwd=ROOT, capture_output=True,
                       text=True, timeout=300)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and not r.stdout


def test_workload_tables():
    wl = bench.workloads()
    for name in ("decode8b", "mixed8b", "longdecode8b", "verify70b", "swa8b", "tiny"):
        make, desc = wl[name]
        assert callable(make) and desc
    (m, n, k), desc = bench.LINEAR_WORKLOADS["linear8b"]
    assert (m, n, k) == (4096, 6144, 4096) and desc


def test_code_digest_ignores_comments_only(tmp_path, monkeypatch):
    csrc = os.path.join(tmp_path, "paper_2609_38981_amd", "csrc")
    os.makedirs(csrc)
    for n in ("vd_attn.hip", "vd_cas.hpp", "vd_hw.hpp"):
        shutil.copy(os.path.join(ROOT, "paper_2609_38981_amd", "csrc", n), csrc)
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    base = bench.kernel_code_digest()
    path = os.path.join(csrc, "vd_cas.hpp")
    with open(path) as f:
        text = f.read()
    with open(path, "w") as f:
        f.write("// a new comment line\n/* and a block\n comment */\n" + text.replace("\n", "\n\n", 3))
    assert bench.kernel_code_digest() == base
    with open(path, "w") as f:
        f.write(text.replace("kTileKeys = 64", "kTileKeys = 32", 1))
    assert bench.kernel_code_digest() != base


def test_measured_traffic_needs_the_same_code(tmp_path, monkeypatch):
    prof = os.path.join(tmp_path, "profiles")
    os.makedirs(prof)
    shutil.copytree(os.path.join(ROOT, "paper_2609_38981_amd", "csrc"),
                    os.path.join(tmp_path, "paper_2609_38981_amd", "csrc"))
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    digest = bench.kernel_code_digest()
    import json

    def write(entries):
        with open(os.path.join(prof, "hbm_traffic.json"), "w") as f:
            json.dump({"entries": entries}, f)

    e = lambda k, w, b, d=digest: dict(kernel=k, workload=w, bytes_per_launch=b, code_sha256=d)
    write([e("split_kernel", "decode8b", 123), e("split_kernel", "longdecode8b", 456),
           e("prefix_kernel", "verify70b", 10), e("split_kernel", "verify70b", 20),
           e("chunk_kernel", "mixed8b", 7, "0" * 64)])
    assert bench.measured_traffic("split_kernel", "decode8b") == 123
    assert bench.measured_traffic("split_kernel", "longdecode8b") == 456
    assert bench.measured_traffic("split_kernel", "mixed8b") is None
    # two kernels of one phase: the sum, only when both are covered
    assert bench.measured_traffic("prefix_kernel+split_kernel", "verify70b") == 30
    assert bench.measured_traffic("prefix_kernel+split_kernel", "decode8b") is None
    # counters taken on other code
    assert bench.measured_traffic("chunk_kernel", "mixed8b") is None
    write([e("split_kernel", "decode8b", 123, "0" * 64)])
    assert bench.measured_traffic("split_kernel", "decode8b") is None


def test_err_vs_gpu():
    ref = np.array([300.0, -1.0, 0.5])
    got = np.array([301.0, -1.0, 0.5])
    e = bench.err_vs_gpu(got, ref)
    assert e["max_abs_err_vs_gpu"] == 1.0
    assert abs(e["max_err_rel_to_max_abs"] - 1.0 / 300.0) < 1e-15
    assert bench.err_vs_gpu(np.zeros(3), np.zeros(3))["max_err_rel_to_max_abs"] == 0.0


def test_cpu_baseline_on_the_tiny_call():
    """The oracle leg on the two-request call: rows rounded to bf16 from the
    oracle's own output differ from it by at most half a bf16 step."""
    call = W.config1()
    sh = call.shape
    kp, vp = call.std_pool(poison=False)
    ref = oracle.paged_attention(call.q_bits(), call.cu_q_lens, call.context_lens, call.page_table,
                                 kp, vp, num_q_heads=sh.num_q_heads, num_kv_heads=sh.num_kv_heads,
                                 head_dim=sh.head_dim, page_size=sh.page_size, window=sh.window)
    bits = W.bf16_bits(ref.astype(np.float32))
    res = bench.cpu_baseline(call, bits, min_seconds=0.05)
    assert res["kind"] == "oracle" and res["unit"] == "GB/s"
    assert res["value"] > 0 and res["cores"] >= 1 and res["sample"]
    scale = float(np.abs(ref).max())
    assert 0 <= res["max_abs_err_vs_gpu"] <= 2.0 ** -8 * scale
