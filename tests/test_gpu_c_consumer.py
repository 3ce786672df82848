"""The C ABI from C: tests/c_consumer.c (built by __graft_entry__.build())
creates a buffer, ingests, samples with the fused gather, checks every gathered
row against the ingested bytes, updates priorities, and round-trips a
checkpoint through host memory, using include/conduit.h and libconduit.so
only."""
import os
import subprocess

import pytest

pytestmark = pytest.mark.gpu

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
BIN = os.path.join(ROOT, "tests", "c_consumer.bin")


def test_c_program_uses_the_abi():
    print("c consumer: create, ingest, sample + gather, update, checkpoint, restore", flush=True)
    assert os.path.exists(BIN), "tests/c_consumer.bin is built by __graft_entry__.build()"
    r = subprocess.run([BIN], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "c consumer ok" in r.stdout
