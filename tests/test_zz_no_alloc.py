"""The compaction entry point that allocates nothing (nsc_compact_noalloc:
tile offsets in the library's static device array) against nsc_compact with
a caller workspace, through the C ABI: index lists and counts bit-identical,
on two calls in a row (the second smaller, so offsets left in the shared
array by the first must not leak into it) and at the size limit."""
import numpy as np
import pytest
import torch

import paper_1703_02529_amd as nsc

pytestmark = pytest.mark.gpu
DEV = "cuda"


def _both(fire_np: np.ndarray):
    n = int(fire_np.size)
    fire = torch.from_numpy(fire_np).to(DEV)
    ws = torch.empty(max(nsc.nsc_compact_workspace_bytes(n), 4), dtype=torch.uint8, device=DEV)
    idx_a = torch.full((max(n, 1),), -7, dtype=torch.int32, device=DEV)
    cnt_a = torch.full((1,), -1, dtype=torch.int32, device=DEV)
    nsc.nsc_compact(fire if n else None, n, idx_a if n else None, cnt_a, ws if n else None)
    idx_b = torch.full((max(n, 1),), -9, dtype=torch.int32, device=DEV)
    cnt_b = torch.full((1,), -2, dtype=torch.int32, device=DEV)
    nsc.nsc_compact_noalloc(fire if n else None, n, idx_b if n else None, cnt_b)
    torch.cuda.synchronize()
    ca, cb = int(cnt_a.item()), int(cnt_b.item())
    want = np.flatnonzero(fire_np)
    assert ca == cb == want.size
    a, b = idx_a.cpu().numpy(), idx_b.cpu().numpy()
    assert np.array_equal(a[:ca], b[:cb])
    assert np.array_equal(b[:cb], want)
    assert (b[cb:] == -9).all(), "entries beyond the count were written"
    return cb


def test_noalloc_equals_workspace_compaction_twice():
    rng = np.random.default_rng(77)
    first = (rng.random(10_000_000) < 0.3).astype(np.uint8)   # 2,442 tiles
    second = (rng.random(12_345) < 0.05).astype(np.uint8)     # 4 tiles, ragged
    print("counts", _both(first), _both(second))
    print("empty", _both(np.zeros(0, np.uint8)), "single", _both(np.ones(1, np.uint8)))


def test_noalloc_at_the_size_limit():
    n = nsc.NSC_NOALLOC_MAX_FLAGS
    fire = np.zeros(n, np.uint8)
    rng = np.random.default_rng(5)
    fire[rng.integers(0, n, 50_000)] = 1
    fire[[0, n - 1]] = 1
    print("count at the limit", _both(fire))
    # one flag more is refused on the host, before any GPU work
    f = torch.zeros(8, dtype=torch.uint8, device=DEV)
    idx = torch.zeros(8, dtype=torch.int32, device=DEV)
    cnt = torch.zeros(1, dtype=torch.int32, device=DEV)
    with pytest.raises(nsc.NscError) as e:
        nsc.nsc_compact_noalloc(f, n + 1, idx, cnt)
    assert e.value.status == nsc.NSC_E_WORKSPACE
