"""bench.py command line on the CPU: the one-GPU contract and the JSON fields
it promises (no GPU needed for either check)."""
import os
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_is_refused_with_a_message():
    res = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"],
                         capture_output=True, text=True, timeout=60)
    assert res.returncode == 2
    assert "one GPU" in res.stderr + res.stdout
    assert res.stdout.strip() == "" or not res.stdout.strip().startswith("{")


def test_record_carries_the_contract_keys():
    src = open(os.path.join(ROOT, "bench.py")).read()
    for key in ('"metric"', '"value"', '"unit"', '"n_gpus"', '"steps"', '"warmup"', '"ms_per_step"',
                '"higher_is_better"', '"scaling"', '"vs_baseline"', '"dtype"', '"data"', '"config"',
                '"roofline"', '"cpu_baseline"'):
        assert key in src, key
    for key in ('"bound"', '"achieved"', '"peak"', '"frac"', '"traffic"'):
        assert key in src, key
