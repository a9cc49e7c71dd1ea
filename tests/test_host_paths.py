"""Host paths of the C ABI on a machine without a GPU: every entry point is
driven with fake, aligned device addresses through its argument checks, its
sort plan and workspace layout, up to its first kernel launch, which fails
(GBA_ERR_HIP) because there is no device.  A workspace one byte short of the
query is refused first (GBA_ERR_WORKSPACE), and no size near the limits
overflows the layout arithmetic.  Run against the host-sanitized build (see
the build module) the same calls check the host code under AddressSanitizer
and UndefinedBehaviorSanitizer.

Nothing here may reach a real GPU with the fake addresses, so the module is
skipped wherever a device is visible."""
import ctypes

import pytest

import paper_2205_11048_amd as gba


def _gpu_visible():
    try:
        import torch
        return torch.cuda.is_available()
    except Exception:   # no torch: no GPU path either
        return False


pytestmark = pytest.mark.skipif(_gpu_visible(), reason="fake device addresses must never reach a GPU")

OK, NULL, INVALID, UNSUPPORTED, WORKSPACE, HIP = 0, 1, 2, 3, 4, 5
P = ctypes.c_void_p
A = 1 << 20          # a fake 16-byte (and 32-byte) aligned "device" address


def fake(i):
    return P(A * (i + 1))


SIZES = [(1, 1, 4, 1), (4095, 7, 16, 3000), (1 << 22, 256, 32, 500_000_000), ((1 << 28) - 1, 4096, 256, 1 << 32),
         (65_536_000, 256, 32, 500_000_000), (10_240_000, 100, 16, 100_000_000)]


def _sparse(L, N, K, D, R, ws_bytes, plan=None):
    args = [fake(0), fake(1), fake(2), K, N, D, R, fake(3), fake(4), 1000, 2, None, 0, 0,
            fake(5), fake(6), fake(7), fake(8), fake(9), fake(10), fake(11), ctypes.c_size_t(ws_bytes)]
    if plan is None:
        return L.gba_aggregate_sparse(*args, fake(12), None)
    return L.gba_aggregate_sparse_plan(*args, plan, fake(12), None)


@pytest.mark.parametrize("N,K,D,R", SIZES)
def test_sparse_host_path(N, K, D, R):
    L = gba.lib()
    for plan in (gba.SORT_AUTO, gba.SORT_PLAIN, gba.SORT_HOT):
        need = gba.gba_aggregate_sparse_plan_workspace_size(N, K, D, R, plan)
        assert need > 0
        assert _sparse(L, N, K, D, R, need - 1, plan) == WORKSPACE
        assert _sparse(L, N, K, D, R, need, plan) == HIP
    assert _sparse(L, N, K, D, R, gba.gba_aggregate_sparse_workspace_size(N, K, D, R)) == HIP


@pytest.mark.parametrize("N,K,D,R", SIZES)
def test_fused_sparse_host_path(N, K, D, R):
    L = gba.lib()
    for opt in ("adagrad", "adam"):
        need = gba.gba_aggregate_apply_sparse_workspace_size(N, K, D, R, opt)
        base = [fake(0), fake(1), fake(2), K, N, D, R, fake(3), fake(4), 1000, 2, None, 0, 0,
                fake(5), fake(6), fake(7), fake(8), None, fake(10)]
        for ws, want in ((need - 1, WORKSPACE), (need, HIP)):
            if opt == "adagrad":
                st = L.gba_aggregate_apply_sparse_adagrad(*base, fake(13), fake(14), 0.01, 1e-8, fake(12),
                                                          ctypes.c_size_t(ws), None, None)
            else:
                st = L.gba_aggregate_apply_sparse_adam(*base, fake(13), fake(14), fake(15), 1e-3, 0.9, 0.999, 1e-8,
                                                       1001, fake(12), ctypes.c_size_t(ws), None, None)
            assert st == want, (opt, ws)


@pytest.mark.parametrize("n,R", [(1, 1), (2049, 1000), (1 << 22, 1 << 24), ((1 << 28) - 1, 1 << 32)])
def test_sort_pull_hash_host_paths(n, R):
    L = gba.lib()
    for plan in (gba.SORT_AUTO, gba.SORT_PLAIN, gba.SORT_HOT):
        need = gba.gba_sort_ids_workspace_size(n, R, plan)
        assert L.gba_sort_ids(fake(0), n, R, plan, fake(1), fake(2), fake(3), ctypes.c_size_t(need - 1), None,
                              None) == WORKSPACE
        assert L.gba_sort_ids(fake(0), n, R, plan, fake(1), fake(2), fake(3), ctypes.c_size_t(need), None,
                              None) == HIP
    need = gba.gba_pull_workspace_size(n, R)
    assert L.gba_pull_rows(fake(0), n, R, fake(1), 32, fake(2), fake(3), fake(4), fake(5), fake(6),
                           ctypes.c_size_t(need - 1), None, None) == WORKSPACE
    assert L.gba_pull_rows(fake(0), n, R, fake(1), 32, fake(2), fake(3), fake(4), fake(5), fake(6),
                           ctypes.c_size_t(need), None, None) == HIP
    need = gba.gba_hash_workspace_size(n)
    cap = 1 << 20
    assert L.gba_hash_find_or_insert(fake(0), fake(1), cap, fake(2), n, fake(3), fake(4), 1 << 19, None, None,
                                     fake(5), ctypes.c_size_t(need - 1), None, None) == WORKSPACE
    assert L.gba_hash_find_or_insert(fake(0), fake(1), cap, fake(2), n, fake(3), fake(4), 1 << 19, None, None,
                                     fake(5), ctypes.c_size_t(need), None, None) == HIP


@pytest.mark.parametrize("P_", [1, 5, 16_000_000, 200_000_000, (1 << 34) + 3])
@pytest.mark.parametrize("K", [1, 256, 4096])
def test_dense_host_paths(P_, K):
    L = gba.lib()
    assert L.gba_aggregate_dense(fake(0), fake(1), K, P_, fake(2), None) == HIP
    assert L.gba_aggregate_apply_dense_adagrad(fake(0), fake(1), K, P_, None, fake(2), fake(3), 0.01, 1e-8,
                                               None) == HIP
    assert L.gba_aggregate_apply_dense_adam(fake(0), fake(1), K, P_, None, fake(2), fake(3), fake(4), 1e-3, 0.9,
                                            0.999, 1e-8, 1001, None) == HIP
    assert L.gba_accumulate_dense(fake(0), fake(1), K, P_, fake(2), None) == HIP
    assert L.gba_finalize_apply_dense_adagrad(fake(0), K, P_, None, fake(2), fake(3), 0.01, 1e-8, 1, None) == HIP
    # the launch count is a host query: one launch unless P spans more than two rounds of resident blocks
    n = ctypes.c_int64(0)
    assert L.gba_aggregate_dense_launches(P_, K, 1, ctypes.byref(n)) == OK
    assert n.value >= 1
    assert L.gba_apply_adagrad(fake(0), fake(1), fake(2), None, None, None, P_, 0, 0, 0.01, 1e-8, None,
                               None) == HIP


def test_row_apply_and_noalloc_host_paths():
    L = gba.lib()
    assert L.gba_apply_adagrad(fake(0), fake(1), fake(2), fake(3), None, fake(4), 1000, 32, 1 << 32, 0.01, 1e-8,
                               None, None) == HIP
    assert L.gba_apply_adam(fake(0), fake(1), fake(2), fake(3), fake(4), None, fake(5), 1000, 32, 1 << 32, 1e-3,
                            0.9, 0.999, 1e-8, 7, None, None) == HIP
    # the no-allocation call: within its array it needs the device (absent here), beyond it it is refused first
    args = [fake(0), fake(1), fake(2), 8, 100_000, 32, 1 << 24, fake(3), fake(4), 1000, 2, None, 0, 0,
            fake(5), fake(6), fake(7), fake(8), fake(9), fake(10), fake(11), None]
    assert L.gba_aggregate_sparse_noalloc(*args) == HIP
    args[4] = 3_000_000
    assert L.gba_aggregate_sparse_noalloc(*args) == gba.ERR_SCRATCH_LIMIT
