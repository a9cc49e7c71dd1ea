"""The measurement kernels (include/gba_ceilings.h) touch exactly the bytes
they are timed for: the read stream folds every word of its input into its
per-wave words once, the copy is exact, and the row gather folds every word
of every listed row once (rows outside the table are skipped)."""
import numpy as np
import pytest
import torch

import paper_2205_11048_amd as gba

pytestmark = pytest.mark.gpu


def _xor_all(a):
    return int(np.bitwise_xor.reduce(np.ascontiguousarray(a).view(np.uint32).reshape(-1))) if a.size else 0


@pytest.mark.parametrize("n_floats,blocks", [(4, 1), (1_000_004, 7), (3 * 2048 * 256 * 4 + 40, 64)])
def test_read_and_copy(n_floats, blocks):
    rng = np.random.default_rng(n_floats)
    h = rng.standard_normal(n_floats).astype(np.float32)
    src = torch.from_numpy(h).cuda()
    sink = torch.full((gba.gba_ceiling_sink_words(blocks),), -1, dtype=torch.int32, device="cuda")
    gba.gba_ceiling_read(src, sink, blocks)
    dst = torch.zeros_like(src)
    gba.gba_ceiling_copy(src, dst, blocks)
    torch.cuda.synchronize()
    assert _xor_all(sink.cpu().numpy()) == _xor_all(h)
    assert torch.equal(dst, src)


@pytest.mark.parametrize("D", [4, 16, 20, 32, 256])
def test_gather_rows(D):
    rng = np.random.default_rng(D)
    R, n = 3001, 50_001
    table = rng.standard_normal((R, D)).astype(np.float32)
    rows = rng.integers(-3, R + 3, n).astype(np.int64)
    sink = torch.full((gba.gba_ceiling_sink_words(37),), -1, dtype=torch.int32, device="cuda")
    gba.gba_ceiling_gather_rows(torch.from_numpy(table).cuda(), torch.from_numpy(rows).cuda(), sink, 37)
    torch.cuda.synchronize()
    ok = rows[(rows >= 0) & (rows < R)]
    assert _xor_all(sink.cpu().numpy()) == _xor_all(table[ok])
