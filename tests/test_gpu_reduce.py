"""GPU unit test of the deferred gradient reduction through the test hook spzt_reduce_jobs.

Each update part reduces the split-K slices of its weight gradients and the column-sum
partials of its bias gradients with one launch over a job list. The kernel's order of
summation is fixed: thread g of `groups` adds slices g, g + groups, ... in turn, then the
group sums are added in g order. The host recomputes every job in exactly that order in
float32 (IEEE additions, as on the device), so outputs must agree bit for bit; columns
between cols and ldo must stay untouched. The job shapes mirror the library's: split-K
slices of a weight gradient (one thread per piece, or eight groups for small outputs
from many slices), column-sum partials (64 groups), the scalar bias sum of the critic
output layer (one column), a ragged job with ld > cols, and an empty job between two
others (the block-to-job map must skip it).
"""
import ctypes

import numpy as np
import pytest

pytestmark = pytest.mark.gpu

# rows, cols, slices, groups, vec, ld, ldo
JOBS = [
    (64, 96, 16, 1, 4, 96, 96),       # split-K slices, one thread per 16-byte piece
    (16, 64, 128, 8, 4, 64, 64),      # small output from many slices: eight groups
    (1, 256, 512, 64, 4, 256, 256),   # column-sum partials
    (0, 32, 7, 1, 4, 32, 32),         # empty job
    (1, 1, 300, 64, 1, 1, 1),         # scalar sum (slice count not a multiple of the groups)
    (3, 12, 5, 2, 4, 16, 20),         # ld > cols, ldo > cols
]


def host_reduce(part, zstride, ld, rows, cols, slices, groups):
    idx = np.arange(rows)[:, None] * ld + np.arange(cols)[None, :]
    sums = []
    for g in range(groups):
        acc = np.zeros((rows, cols), np.float32)
        for z in range(g, slices, groups):
            acc = (acc + part[z * zstride + idx]).astype(np.float32)
        sums.append(acc)
    tot = sums[0]
    for g in range(1, groups):
        tot = (tot + sums[g]).astype(np.float32)
    return tot


@pytest.fixture(scope="module")
def hook():
    torch = pytest.importorskip("torch")
    from paper_2312_06126_amd import spz
    lib = spz.load()
    f = lib.spzt_reduce_jobs
    PP, P64, P32 = ctypes.POINTER(ctypes.c_void_p), ctypes.POINTER(ctypes.c_int64), ctypes.POINTER(ctypes.c_int32)
    f.argtypes = [ctypes.c_int32, PP, PP, P64, P64, P64, P32, P32, P32, P32, P32]
    f.restype = ctypes.c_int
    return torch, f


def run(torch, f, jobs):
    n = len(jobs)
    arr = lambda t, v: (t * n)(*v)
    parts, outs = [], []
    for rows, cols, slices, groups, vec, ld, ldo in jobs:
        zs = max(rows, 1) * ld
        parts.append(torch.randn(slices * zs + 64, dtype=torch.float32, device="cuda"))
        outs.append(torch.full((max(rows, 1) * ldo + 8,), float("nan"), dtype=torch.float32, device="cuda"))
    rc = f(n, arr(ctypes.c_void_p, [p.data_ptr() for p in parts]), arr(ctypes.c_void_p, [o.data_ptr() for o in outs]),
           arr(ctypes.c_int64, [max(j[0], 1) * j[5] for j in jobs]), arr(ctypes.c_int64, [j[5] for j in jobs]),
           arr(ctypes.c_int64, [j[6] for j in jobs]), arr(ctypes.c_int32, [j[0] for j in jobs]),
           arr(ctypes.c_int32, [j[1] for j in jobs]), arr(ctypes.c_int32, [j[2] for j in jobs]),
           arr(ctypes.c_int32, [j[3] for j in jobs]), arr(ctypes.c_int32, [j[4] for j in jobs]))
    return rc, [p.cpu().numpy() for p in parts], [o.cpu().numpy() for o in outs]


def test_reduce_jobs_match_host_order_bit_for_bit(hook):
    torch, f = hook
    torch.manual_seed(0)
    rc, parts, outs = run(torch, f, JOBS)
    assert rc == 0
    for (rows, cols, slices, groups, vec, ld, ldo), part, out in zip(JOBS, parts, outs):
        if rows == 0:
            assert np.all(np.isnan(out))
            continue
        ref = host_reduce(part, rows * ld, ld, rows, cols, slices, groups)
        got = out[: rows * ldo].reshape(rows, ldo)
        assert np.array_equal(got[:, :cols].view(np.uint32), ref.view(np.uint32)), (rows, cols, slices, groups)
        assert np.all(np.isnan(got[:, cols:])) and np.all(np.isnan(out[rows * ldo:]))


@pytest.mark.parametrize("bad", [(8, 6, 4, 1, 4, 8, 8),      # cols not a multiple of the vector width
                                 (8, 8, 4, 3, 4, 8, 8),      # groups not a power of two
                                 (8, 8, 0, 1, 4, 8, 8),      # no slices
                                 (8, 8, 4, 1, 2, 8, 8)])     # vector width other than 1 or 4
def test_reduce_jobs_refuse_bad_jobs(hook, bad):
    torch, f = hook
    rc, _, _ = run(torch, f, [JOBS[0], bad])
    assert rc == -1
