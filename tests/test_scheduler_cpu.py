"""Copy-scheduler tests on the CPU: the host-side Prefetcher driven by a copy
engine with a simulated clock (tests/cpp/test_scheduler.cpp, built with g++ and
the address/undefined-behaviour sanitizers)."""
import json
import os
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)


@pytest.fixture(scope="module")
def binary(tmp_path_factory):
    out = str(tmp_path_factory.mktemp("sched") / "test_scheduler")
    cmd = ["g++", "-std=c++17", "-O1", "-g", "-fsanitize=address,undefined", "-fno-omit-frame-pointer",
           os.path.join(HERE, "cpp", "test_scheduler.cpp"),
           os.path.join(ROOT, "paper_2410_22134_amd", "csrc", "scheduler.cpp"), "-o", out]
    subprocess.run(cmd, check=True)
    return out


def test_scheduler_unit_tests(binary):
    r = subprocess.run([binary], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "ALL OK" in r.stdout


def test_paper_chunk_preemption_example(binary):
    g = json.load(open(os.path.join(HERE, "golden", "chunk_preemption_example.json")))
    r = subprocess.run([binary, "example"], capture_output=True, text=True, timeout=60, check=True)
    chunked, unchunked, early = (float(v) for v in r.stdout.split())
    # times are in units of one chunk copy
    # chunked: the miss waits for the chunk in progress (the second) and starts at its end
    assert chunked == g["high_starts_after_chunk_with_chunking"] + 1
    # unchunked: it waits for the whole expert (all three chunks)
    assert unchunked == g["chunks_per_expert"]
    # early preemption: the miss is known while the first chunk copies, so it goes
    # before the second chunk
    assert early == g["early_preemption_high_starts_before_chunk"]
