"""Host logic of bench.py (no GPU): the one-GPU contract, the gate that keeps
a committed counter summary out of the JSON line once the kernel sources
differ from the ones it was taken on, and the workloads the encoder's
instruction count applies to."""

import hashlib
import os
import subprocess
import sys

import bench
import dq_workloads as wlmod
from conftest import ROOT


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode != 0
    assert "--gpus 2" in r.stderr
    assert r.stdout.strip() == ""


def test_summary_is_used_only_for_the_sources_it_was_taken_on(tmp_path):
    src = tmp_path / "kernel.hip"
    src.write_text("// kernel v1\n")
    digest = hashlib.sha256(src.read_bytes()).hexdigest()
    summary = tmp_path / "summary.md"
    summary.write_text(f"| SQ_INSTS_VALU | 1,234 | 5 |\n\n    kernel_source_sha256: {digest}\n")
    assert bench._summary_text(str(summary), [str(src)]) is not None
    src.write_text("// kernel v2\n")
    assert bench._summary_text(str(summary), [str(src)]) is None
    assert bench._summary_text(str(tmp_path / "missing.md"), [str(src)]) is None


def test_encoder_figure_applies_to_the_summarized_coding_only():
    for name in ("b16_t32k", "b64_t8k", "b1_t128k"):
        wl = wlmod.workload(name)
        assert bench.encode_valu_per_stream(wl, "literal") is None
    for name, variant in (("b16_t32k", "literal"), ("b32_t32k_g8", "paper"), ("b16_t32k_tok", "paper")):
        assert bench.encode_valu_per_stream(wlmod.workload(name, variant), variant) is None
    assert bench.encode_valu_per_stream(wlmod.workload("b1_t128k", "paper", 3.0), "paper") is None
    a = bench.encode_valu_per_stream(wlmod.workload("b16_t32k"), "paper")
    b = bench.encode_valu_per_stream(wlmod.workload("b64_t8k"), "paper")
    assert a == b                      # same coding: the same per-stream figure, or both None
    assert a is None or 500 < a < 20000


def test_cpu_baseline_uses_a_pool_of_host_cores(monkeypatch):
    monkeypatch.setattr(bench, "CPU_SECONDS", 0.5)
    for name in ("b1_t4k", "b1_t4k_tok"):
        r = bench.cpu_baseline(wlmod.workload(name), 0)
        assert r["kind"] == "oracle" and r["unit"] == "tokens/s" and r["value"] > 0
        assert r["cores"] == bench._pool_size() and 1 <= r["cores"] <= 16
        assert f"{r['cores']} single-threaded processes" in r["sample"]


def test_paper_context_quotes_the_papers_hardware():
    c = bench.PAPER_CONTEXT
    assert "H20" in c["hardware"]
    assert c["decode_tokens_per_s"]["d_quant"] == 563.6 and c["decode_tokens_per_s"]["bf16"] == 159.5
    assert c["throughput_gain"] == 3.5 and c["peak_memory_gib"]["d_quant_batch_128_8k_prompt"] == 49.4
