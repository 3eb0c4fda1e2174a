"""Host logic of bench.py, on the CPU: the kernel-source fingerprint that
gates the committed HBM-traffic figure, the lookup of that figure, the
one-GPU guard, the workload table against the five measured configurations,
and the algorithmic byte count of the 1M full-context call."""
import os
import re
import subprocess
import sys

import bench
from paper_2607_21535_amd import inputs as I

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_fingerprint_ignores_comments_and_spacing():
    a = "int f(int x) {\n  // note\n  return x + 1;  /* block\n   note */\n}\n"
    b = "int f(int x) { return x + 1; }"
    assert bench._code_only(a) == bench._code_only(b)
    assert bench._code_only(a) != bench._code_only(b.replace("+ 1", "+ 2"))


def test_fingerprint_is_stable_hex():
    h = bench.kernel_source_hash()
    assert re.fullmatch(r"[0-9a-f]{16}", h)
    assert h == bench.kernel_source_hash()


def test_traffic_is_read_only_for_the_current_source(tmp_path, monkeypatch):
    p = tmp_path / "traffic.txt"
    monkeypatch.setattr(bench, "PROFILE_TRAFFIC", str(p))
    p.write_text(f"kernel_source_sha256_16: {bench.kernel_source_hash()}\n"
                 "hbm_bytes_per_attention_call: 2157370878\n")
    assert bench.profiled_traffic("draft_loop_s1m") == 2157370878.0
    assert bench.profiled_traffic("draft_loop_s128k") is None  # taken for the 1M loop only
    p.write_text("kernel_source_sha256_16: 0123456789abcdef\nhbm_bytes_per_attention_call: 1\n")
    assert bench.profiled_traffic("draft_loop_s1m") is None  # another kernel source
    p.write_text(f"kernel_source_sha256_16: {bench.kernel_source_hash()}\n")
    assert bench.profiled_traffic("draft_loop_s1m") is None  # no figure
    os.remove(p)
    assert bench.profiled_traffic("draft_loop_s1m") is None  # no summary


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, "bench.py", "--gpus", "2"], cwd=ROOT, capture_output=True,
                       text=True, timeout=300)
    assert r.returncode == 2
    assert "one GPU" in r.stderr and r.stdout == ""


def test_workloads_are_the_five_configurations():
    w = I.WORKLOADS
    c0, c1, c2, c3, c4 = (w[n] for n in ("decode_s8k", "draft_loop_s128k", "draft_loop_s1m",
                                           "batch32_varlen", "ring_b8"))
    assert (c0.B, c0.Hq, c0.Hkv, c0.d, c0.S, c0.W, c0.sink, c0.gamma) == (1, 16, 2, 128, 8192, 512, 4, 1)
    assert (c1.B, c1.Hq, c1.Hkv, c1.d, c1.S, c1.W, c1.sink, c1.gamma) == (1, 16, 2, 256, 131072, 2048, 4, 3)
    assert (c2.B, c2.Hq, c2.Hkv, c2.d, c2.S, c2.W, c2.sink, c2.gamma) == (1, 32, 2, 256, 1 << 20, 2048, 4, 7)
    assert (c2.sink_bias, c2.bias_rows) == (4.0, 4)
    assert (c3.B, c3.Hq, c3.Hkv, c3.d, c3.S_lo, c3.S, c3.W, c3.sink) == (32, 32, 2, 256, 65536, 1 << 20, 2048, 4)
    assert (c4.B, c4.Hq, c4.Hkv, c4.d, c4.W, c4.sink, c4.R_w) == (8, 32, 2, 256, 2048, 4, 2048)
    assert (c4.iterations, c4.max_accept) == (1000, 8)
    assert len({x.seed for x in w.values()}) == len(w)
    for x in w.values():
        assert x.scale == 1.0 / x.d ** 0.5


def test_algorithmic_bytes_of_the_1m_call():
    wl = I.WORKLOADS["draft_loop_s1m"]
    # 2048 bytes of K and V per token at d = 256 with two KV heads (the
    # per-token size Section 3 gives for a Qwen draft layer), 2 GiB at 1M
    # tokens, plus q and the output
    assert wl.Hkv * wl.d * 2 * 2 == 2048
    assert bench.full_call_bytes(wl) == 2 * 2**30 + 2 * 32 * 256 * 2 == 2147516416
