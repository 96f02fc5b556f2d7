"""Host-only checks of logic around the kernels: the bench refuses more than one GPU, and the
default split plan never launches more parts than a batch has 64-token blocks."""

import os
import subprocess
import sys
import types

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_bench_refuses_several_gpus():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=300, cwd=ROOT)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


@pytest.fixture
def sm(monkeypatch):
    if not os.path.exists(os.path.join(ROOT, "paper_2602_10718_amd", "libsnapmla.so")):
        pytest.fail("libsnapmla.so is not built (run __graft_entry__.build())")
    from paper_2602_10718_amd import snapmla
    props = types.SimpleNamespace(multi_processor_count=256)
    monkeypatch.setattr(snapmla.torch.cuda, "get_device_properties", lambda *a, **k: props)
    monkeypatch.setattr(snapmla.torch.cuda, "current_device", lambda: 0)
    return snapmla


@pytest.mark.parametrize("q_len,H,blocks,expect", [
    (1, 64, None, 256),       # one row group: one part per CU
    (1, 128, None, 128),      # two row groups
    (2, 128, None, 64),       # four row groups
    (1, 16, 20592, 256),      # the headline batch: no cap
    (1, 16, 4, 8),            # a 4-block batch: at least 8 parts, no more
    (1, 64, 100, 104),        # capped at the blocks, rounded up to 8
    (2, 128, 30, 32),
])
def test_default_num_splits(sm, q_len, H, blocks, expect):
    assert sm.default_num_splits(q_len, H, total_blocks=blocks) == expect
