"""bench.py's host side, without a GPU: more than one GPU is refused before
anything touches a device, the FLOP count is the standard attention count
(4 d per visible query-key pair), and the oracle baseline reports what the
bench line promises."""
import subprocess
import sys
from pathlib import Path

import pytest

import bench
import workloads as W

ROOT = Path(__file__).resolve().parents[1]


def test_more_than_one_gpu_exits_with_a_message():
    r = subprocess.run([sys.executable, str(ROOT / "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120, cwd=ROOT)
    assert r.returncode != 0
    assert "--gpus 1" in r.stderr and r.stdout == ""


@pytest.mark.parametrize("name,flops", [
    ("bert_l128", 4 * 64 * 12 * 128 * 128),
    ("dec_l4096", 4 * 128 * 4 * 32 * 4096 * 4097 // 2),
    ("long_l32768", 4 * 128 * 32 * 32768 * 32769 // 2),
])
def test_flop_count(name, flops):
    assert W.WORKLOADS[name].flops == pytest.approx(flops, rel=1e-12)


def test_cpu_baseline_record():
    """The oracle leg times whole heads of the bench's own seeded tensors and
    names the BLAS it ran on."""
    w = W.WORKLOADS["bert_l128"]
    inp = W.make_inputs(w)
    rec = bench.cpu_baseline(w, inp, target_s=0.2)
    assert rec["kind"] == "oracle" and rec["unit"] == "TFLOP/s"
    assert rec["value"] > 0 and rec["cores"] >= 1 and rec["affinity_cores"] >= 1
    assert "heads of the same seeded tensors" in rec["sample"] and rec["seconds"] > 0
    assert 1 <= rec["heads"] <= w.B * w.H
    assert rec["blas"] and "not reported" not in rec["blas"]


def test_percentile_and_bytes():
    assert bench.percentile([5, 1, 4, 2, 3], 50) == 3
    assert bench.percentile([5, 1, 4, 2, 3], 10) == 1 and bench.percentile([1, 2, 3], 90) == 3
    w = W.WORKLOADS["dec_l4096"]
    # Q, K, V read and O written once in bf16, 5 bytes of resid and flags per row
    assert bench.w_bytes(w) == 4 * 32 * (4 * 4096 * 128 * 2) + 5 * 4 * 32 * 4096


def test_kernel_hash_is_the_source_hash():
    import hashlib
    src = (ROOT / "paper_2507_16676_amd" / "csrc" / "fabft_kernels.hip").read_bytes()
    assert bench.kernel_src_sha() == hashlib.sha256(src).hexdigest()[:16]
