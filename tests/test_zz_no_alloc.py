"""GPU: the allocation-free entry point (tri_residual_rmsnorm_noalloc, through
the C ABI via the binding) against the ordinary entry point
(tri_residual_rmsnorm) on the same inputs: two calls in a row, the second
with fewer rows, for a split version (its partial sums through the GPU's
fixed scratch instead of the version's own) and for a one-workgroup-per-row
version. Both entry points run the same kernel with the same reduction
order, so outputs must agree bit for bit; each output is also checked
against the CPU oracle. Each case prints its name before touching the GPU.
"""
import numpy as np
import pytest
import torch

from oracle import numerics as nm
from oracle import ops as O
from oracle import selection as S
from tests.parity import check
import workloads as wl

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


@pytest.fixture(scope="module")
def tri():
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2609_37241_amd as tri
    return tri


@pytest.mark.parametrize("dtype,H,rows,variant", [
    (nm.BF16, 65536, (8, 5), S.RN_SPLIT),      # 4 workgroups per row; bucket 3
    (nm.F32, 32772, (6, 5), S.RN_SPLIT),       # 5 per row, the last one ragged; bucket 3
    (nm.BF16, 4096, (4, 3), S.RN_BLOCK[2]),    # one workgroup per row; bucket 2
])
def test_noalloc_entry_equals_the_ordinary_entry(tri, dtype, H, rows, variant):
    print(f"no-alloc entry: {dtype} H={H} rows={rows}", flush=True)
    r = np.random.Generator(np.random.PCG64(H + rows[0]))
    w = wl.host_weight(r, H, dtype)
    wd = wl.to_torch(w, dtype, DEV)
    cache = tri.SpecCache()
    try:
        for T in rows:                         # both in one token bucket: one version
            x, res = wl.host_array(r, (T, H), dtype), wl.host_array(r, (T, H), dtype)
            xd, rd = wl.to_torch(x, dtype, DEV), wl.to_torch(res, dtype, DEV)
            y1, ro1 = cache.residual_rmsnorm(xd, rd, wd, 1e-6)    # installs on the first row count
            sel1 = cache.last_selection().as_tuple()
            y2, ro2 = torch.empty_like(xd), torch.empty_like(xd)
            cache.residual_rmsnorm_noalloc(xd, rd, wd, 1e-6, out=y2, residual_out=ro2)
            sel2 = cache.last_selection().as_tuple()
            torch.cuda.synchronize()
            assert sel2 == sel1 and sel2[3] == variant
            check(f"T={T} y", wl.from_torch(y2), wl.from_torch(y1), dtype, exact=True)
            check(f"T={T} res_out", wl.from_torch(ro2), wl.from_torch(ro1), dtype, exact=True)
            wy, wh = O.residual_rmsnorm(x, res, w, 1e-6, dtype)
            check(f"T={T} y vs oracle", wl.from_torch(y2), wy, dtype)
            check(f"T={T} res_out vs oracle", wl.from_torch(ro2), wh, dtype, exact=True)
        assert cache.stats()["n_versions"] == 1
    finally:
        torch.cuda.synchronize()
        cache.close()


def test_noalloc_entry_misses_without_installing(tri):
    print("no-alloc entry: miss", flush=True)
    cache = tri.SpecCache(auto_install=True)
    try:
        x = torch.ones((2, 65536), dtype=torch.bfloat16, device=DEV)
        w = torch.ones(65536, dtype=torch.bfloat16, device=DEV)
        y, ro = torch.empty_like(x), torch.empty_like(x)
        with pytest.raises(tri.TriError) as e:
            cache.residual_rmsnorm_noalloc(x, x, w, out=y, residual_out=ro)
        assert e.value.status == tri.MISS
        assert cache.stats()["n_versions"] == 0
    finally:
        torch.cuda.synchronize()
        cache.close()
