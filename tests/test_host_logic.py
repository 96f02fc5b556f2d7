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


@pytest.mark.parametrize("lens,q_len,H,kv,expect", [
    ([256], 1, 16, "e4m3", True),                 # 4 blocks on 8 parts: one piece, no combine
    ([1024] * 256, 1, 64, "e4m3", True),          # every sequence one part's worth, 256 workgroups
    ([1024] * 257, 1, 64, "e4m3", False),         # more workgroups than CUs
    ([4096] * 32, 1, 64, "e4m3", False),          # 64 blocks per sequence against 8 per part
    ([256], 1, 128, "e4m3", False),               # two row groups: no direct rows in the FP8 decode
    ([256], 1, 128, "bf16", True),                # the BF16 decode writes them with any row count
    ([64 * 4, 64], 1, 64, "e4m3", True),          # 4 blocks against 5/8 + 4
    ([64 * 4 + 1, 64], 1, 64, "e4m3", False),     # 5 blocks against 6/8 + 4: beyond the slack
])
def test_prefer_unsplit(sm, lens, q_len, H, kv, expect):
    from paper_2602_10718_amd import runner
    assert runner.prefer_unsplit(lens, q_len, H, kv) == expect
