"""GPU: the read-stream ceiling kernel (snapmla_debug_read_ceiling) reads every listed page, and the
plain read stream (snapmla_debug_read_stream) reads every word of its buffer.

The kernel is a measurement tool: it streams pages into LDS with the decode's copy
structure and folds the first KiB of every latent and RoPE page into a per-unit XOR.
The checksums are compared with the same XOR formed on the host from the cache bytes
(random pages, so a missed, repeated or misplaced page changes the result), for
ranges of one block, of a few blocks and of the largest allowed size, an id outside
the pool (read as page 0) and an empty list.
"""

import numpy as np
import pytest
import torch

from paper_2602_10718_amd import snapmla as sm

pytestmark = pytest.mark.gpu


def _expected(lat, rope, pages, units, num_pages):
    first_lat = lat.reshape(lat.shape[0], -1)[:, :1024].view(np.uint32)       # [P][256]
    first_rope = rope.reshape(rope.shape[0], -1)[:, :512].view(np.uint32)     # 1 KiB of bf16 -> [P][256]
    n = len(pages)
    out = np.zeros(units, np.uint32)
    for u in range(units):
        gs, ge = u * n // units, (u + 1) * n // units
        acc = np.uint32(0)
        for p in pages[gs:ge]:
            p = p if 0 <= p < num_pages else 0
            acc ^= np.bitwise_xor.reduce(first_lat[p] ^ first_rope[p])
        out[u] = acc
    return out


def _run(lat, sc, rope, pages, units):
    lat_d = torch.from_numpy(lat).cuda()
    sc_d = torch.from_numpy(sc).cuda()
    rope_d = torch.from_numpy(rope.view(np.int16)).cuda()
    pages_d = torch.from_numpy(np.asarray(pages, np.int32)).cuda()
    out = torch.full((units,), -1, dtype=torch.int32, device="cuda")
    print(f"[read_ceiling] pages={len(pages)} units={units}", flush=True)
    sm.snapmla_debug_read_ceiling(lat_d, sc_d, rope_d, pages_d, lat.shape[0], units, out)
    torch.cuda.synchronize()
    return out.cpu().numpy().view(np.uint32)


@pytest.mark.parametrize("nblk,units", [(1, 1), (7, 3), (50, 50), (300, 4), (1792, 1), (3000, 2)])
def test_checksums_match_host(nblk, units):
    rng = np.random.default_rng(nblk * 7 + units)
    P = 97
    lat = rng.integers(0, 256, (P, 64, 512), dtype=np.uint8)
    sc = rng.standard_normal((P, 64)).astype(np.float32)
    rope = rng.integers(0, 1 << 16, (P, 64, 64), dtype=np.uint16)
    pages = rng.integers(0, P, nblk).astype(np.int32)
    got = _run(lat, sc, rope, pages, units)
    assert np.array_equal(got, _expected(lat, rope, pages, units, P))


def test_out_of_range_ids_read_page_zero_and_empty_list():
    rng = np.random.default_rng(5)
    P = 16
    lat = rng.integers(0, 256, (P, 64, 512), dtype=np.uint8)
    sc = rng.standard_normal((P, 64)).astype(np.float32)
    rope = rng.integers(0, 1 << 16, (P, 64, 64), dtype=np.uint16)
    pages = np.array([3, -1, 16, 1 << 30, 5], np.int32)
    got = _run(lat, sc, rope, pages, 2)
    assert np.array_equal(got, _expected(lat, rope, pages, 2, P))
    empty = _run(lat, sc, rope, np.zeros(0, np.int32), 3)
    assert np.array_equal(empty, np.zeros(3, np.uint32))


@pytest.mark.parametrize("words,grid", [(1, 1), (1000, 3), (256 * 7 + 5, 2), (1 << 18, 64)])
def test_plain_stream_checksums(words, grid):
    rng = np.random.default_rng(words + grid)
    buf = rng.integers(0, 1 << 32, (words, 4), dtype=np.uint32)
    out = torch.full((grid,), -1, dtype=torch.int32, device="cuda")
    print(f"[read_stream] words={words} grid={grid}", flush=True)
    sm.snapmla_debug_read_stream(torch.from_numpy(buf.view(np.int32)).cuda(), grid, out)
    torch.cuda.synchronize()
    got = out.cpu().numpy().view(np.uint32)
    # thread t of workgroup g reads words (g + grid * j) * 256 + t
    owner = (np.arange(words) // 256) % grid
    folded = np.bitwise_xor.reduce(buf, axis=1)
    exp = np.array([np.bitwise_xor.reduce(folded[owner == g]) if np.any(owner == g) else 0 for g in range(grid)],
                   np.uint32)
    assert np.array_equal(got, exp)
