"""Host logic of bench.py, on the CPU: the run refuses more than one GPU
before touching any device, and the HBM traffic it reports for a kernel
comes from the committed rocprofv3 counter summary only when that summary
was taken on the same workload and on the kernel's current GEMM source."""

import hashlib
import os
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)

import bench  # noqa: E402

SPEECH = "speech_440_2048x4_1973_sigmoid_b16384"


def test_more_than_one_gpu_is_refused():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120)
    assert r.returncode == 2
    assert "exactly one GPU" in r.stderr
    assert r.stdout.strip() == ""


def fake_tree(tmp_path, workload, fp32_src, bf16_src, sha32=None, sha16=None):
    (tmp_path / "profiles").mkdir()
    csrc = tmp_path / "paper_1606_00511_amd" / "csrc"
    csrc.mkdir(parents=True)
    (csrc / "gemm.hip").write_bytes(fp32_src)
    (csrc / "gemm_bf16.hip").write_bytes(bf16_src)
    sha32 = sha32 or hashlib.sha256(fp32_src).hexdigest()
    sha16 = sha16 or hashlib.sha256(bf16_src).hexdigest()
    (tmp_path / "profiles" / "speech_b16384_hbm_counters.md").write_text(
        "table above\n\n```\n"
        "workload %s\n"
        "traffic_bytes_per_launch hf_gemm_rfwd 1.5e+09\n"
        "traffic_bytes_per_launch hf_hgemm_rfwd 4.0e+08\n"
        "gemm_source_sha256 %s\n"
        "gemm_bf16_source_sha256 %s\n```\n" % (workload, sha32, sha16))


def test_counter_traffic_rules(tmp_path, monkeypatch):
    fake_tree(tmp_path, SPEECH, b"fp32 source", b"bf16 source")
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    assert bench.counter_traffic("hf_gemm_rfwd", SPEECH) == 1.5e9
    assert bench.counter_traffic("hf_hgemm_rfwd", SPEECH) == 4.0e8
    # another workload, or a kernel the summary does not cover
    assert bench.counter_traffic("hf_gemm_rfwd", "mnist_784_100_10_sigmoid_b1000") is None
    assert bench.counter_traffic("hf_gemm_wgrad", SPEECH) is None


@pytest.mark.parametrize("stale", ["fp32", "bf16"])
def test_counter_traffic_needs_the_current_source(tmp_path, monkeypatch, stale):
    fake_tree(tmp_path, SPEECH, b"fp32 source", b"bf16 source",
              sha32="0" * 64 if stale == "fp32" else None,
              sha16="0" * 64 if stale == "bf16" else None)
    monkeypatch.setattr(bench, "ROOT", str(tmp_path))
    f32 = bench.counter_traffic("hf_gemm_rfwd", SPEECH)
    b16 = bench.counter_traffic("hf_hgemm_rfwd", SPEECH)
    assert (f32 is None) == (stale == "fp32")
    assert (b16 is None) == (stale == "bf16")


def test_committed_summary_matches_the_sources():
    """The committed summary names the speech workload; whether its hashes
    are current is what the traffic field of a bench line shows."""
    text = open(os.path.join(ROOT, "profiles", "speech_b16384_hbm_counters.md")).read()
    assert ("workload %s" % SPEECH) in text
    assert "traffic_bytes_per_launch hf_gemm_rfwd" in text
