"""The C ABI library loads and exports every entry point its header declares
(CPU only: nothing here launches a kernel)."""
import ctypes
import os
import re

import pytest

import paper_2205_11048_amd as gba

INCLUDE = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include")


def declared_functions():
    names = set()
    for h in sorted(os.listdir(INCLUDE)):
        if not h.endswith(".h"):
            continue
        text = open(os.path.join(INCLUDE, h)).read()
        text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
        names |= set(re.findall(r"^\s*(?:const\s+)?\w[\w\s\*]*?\b(gba_\w+)\s*\(", text, flags=re.M))
    return sorted(names)


def test_header_declares_the_five_calls():
    names = declared_functions()
    for n in ("gba_token_weights", "gba_aggregate_dense", "gba_aggregate_sparse",
              "gba_apply_adagrad", "gba_apply_adam"):
        assert n in names


def test_library_exports_every_declared_symbol():
    if not os.path.exists(gba.LIB_PATH):
        pytest.fail("libgba.so is not built (python -m paper_2205_11048_amd.build)")
    L = ctypes.CDLL(gba.LIB_PATH)
    for n in declared_functions():
        assert hasattr(L, n), n


def test_status_strings_and_workspace_query():
    L = gba.lib()
    assert L.gba_status_string(0) == b"ok"
    assert b"workspace" in L.gba_status_string(4)
    # pure host queries: sizes grow with N and D, bad widths are refused
    a = gba.gba_aggregate_sparse_workspace_size(1000, 4, 16, 10_000)
    b = gba.gba_aggregate_sparse_workspace_size(100_000, 4, 16, 10_000)
    c = gba.gba_aggregate_sparse_workspace_size(100_000, 4, 64, 10_000)
    assert 0 < a < b < c
    assert gba.gba_aggregate_sparse_workspace_size(0, 1, 4, 1) > 0
    for bad in [(10, 4, 6, 100), (10, 4, 260, 100), (10, 0, 8, 100), (10, 5000, 8, 100),
                (10, 4, 8, 0), (-1, 4, 8, 100), (10, 4, 8, (1 << 32) + 1)]:
        with pytest.raises(gba.GBAError):
            gba.gba_aggregate_sparse_workspace_size(*bad)


def test_host_checks_return_before_any_launch():
    L = gba.lib()
    # the no-allocation sparse call refuses sizes beyond its fixed array before
    # any device work (D = 256 just above 2^20 occurrences)
    assert b"no-allocation" in L.gba_status_string(6)
    assert gba.gba_aggregate_sparse_workspace_size(1_100_000, 4, 256, 1000) > gba.NOALLOC_SCRATCH_BYTES
    assert L.gba_aggregate_sparse_noalloc(None, None, None, 4, 1_100_000, 256, 1000, None, None, 0, 0, None, 0, 0,
                                          None, None, None, None, None, None, None, None) == 6
    assert L.gba_aggregate_sparse_noalloc(None, None, None, 0, 10, 16, 1000, None, None, 0, 0, None, 0, 0,
                                          None, None, None, None, None, None, None, None) == 2
    assert L.gba_aggregate_sparse_noalloc(None, None, None, 4, 10, 6, 1000, None, None, 0, 0, None, 0, 0,
                                          None, None, None, None, None, None, None, None) == 3
    # null pointers and bad sizes are refused on the host, without touching a GPU
    assert L.gba_token_weights(None, 4, 0, 0, None, None, None, None, None) == 1
    assert L.gba_token_weights(None, 0, 0, 0, None, None, None, None, None) == 1
    assert L.gba_aggregate_dense(None, None, 0, 10, None, None) == 2
    assert L.gba_aggregate_dense(None, None, 3, 0, None, None) == 0
    assert L.gba_apply_adagrad(None, None, None, None, None, None, 0, 0, 0, 0.1, 0.0, None, None) == 0
    assert L.gba_apply_adam(None, None, None, None, None, None, None, 10, 0, 0, 0.1, 0.9, 0.999, 0.0, 0,
                            None, None) == 2


def test_dense_launch_query_host_checks():
    L = gba.lib()
    assert L.gba_aggregate_dense_launches(10, 3, 0, None) == 1
    for bad in [(10, 0, 0), (-1, 3, 0), (10, 3, 4), (10, 3, -1)]:
        with pytest.raises(gba.GBAError):
            gba.gba_aggregate_dense_launches(*bad)
    assert gba.gba_aggregate_dense_launches(0, 3) == 0


def test_token_of_batch_host_function():
    """The token rule is a host function of the library: no GPU needed."""
    import oracle
    for M in (1, 4, 32):
        for i in (0, 1, M - 1, M, 5 * M + 2):
            assert gba.gba_token_of_batch(i, M) == oracle.token_of_batch(i, M)
    assert gba.gba_token_of_batch(-1, 4) == -1 and gba.gba_token_of_batch(3, 0) == -1


def test_sort_workspace_query_and_host_checks():
    L = gba.lib()
    # the hot-key plan needs a third key/index array pair; where the key width
    # leaves it no room (8-bit or 32-bit keys) it is the plain plan
    n = 5_000_000
    plain = gba.gba_sort_ids_workspace_size(n, 500_000_000, gba.SORT_PLAIN)
    hot = gba.gba_sort_ids_workspace_size(n, 500_000_000, gba.SORT_HOT)
    assert hot >= plain + 8 * n
    assert gba.gba_sort_ids_workspace_size(n, 500_000_000, gba.SORT_AUTO) == hot
    assert gba.gba_sort_ids_workspace_size(1000, 500_000_000, gba.SORT_AUTO) == \
        gba.gba_sort_ids_workspace_size(1000, 500_000_000, gba.SORT_PLAIN)
    for R in (200, 1 << 32):
        assert gba.gba_sort_ids_workspace_size(n, R, gba.SORT_HOT) == gba.gba_sort_ids_workspace_size(n, R, 0)
    for bad in [(-1, 10, 0), (10, 0, 0), (10, (1 << 32) + 1, 0), (10, 10, 2), (10, 10, -2)]:
        with pytest.raises(gba.GBAError):
            gba.gba_sort_ids_workspace_size(*bad)
    assert L.gba_sort_ids(None, 10, 100, 0, None, None, None, 0, None, None) == 1
    assert L.gba_sort_ids(None, 10, 100, 5, None, None, None, 0, None, None) == 2


def test_fused_sparse_host_checks():
    L = gba.lib()
    # a missing table with occurrences to apply is refused before any launch
    assert L.gba_aggregate_apply_sparse_adagrad(None, None, None, 3, 10, 32, 100, None, None, 0, 0, None, 0, 0,
                                                None, None, None, None, None, None, None, None, 0.1, 0.0, None, 0,
                                                None, None) == 1
    assert L.gba_aggregate_apply_sparse_adam(None, None, None, 3, 10, 32, 100, None, None, 0, 0, None, 0, 0, None,
                                             None, None, None, None, None, None, None, None, 0.1, 1.5, 0.9, 0.0, 1,
                                             None, 0, None, None) == 2
    with pytest.raises(gba.GBAError):
        gba.gba_aggregate_apply_sparse_workspace_size(10, 0, 32, 100, "adagrad")
    with pytest.raises(gba.GBAError):
        gba.gba_aggregate_apply_sparse_workspace_size(10, 3, 32, 100, 3)
    # the rows are applied in the row pass for Adagrad at 20-32 floats; else the means need room
    n = 100_000
    plain = gba.gba_aggregate_sparse_workspace_size(n, 3, 32, 1000)
    assert gba.gba_aggregate_apply_sparse_workspace_size(n, 3, 32, 1000, "adagrad") == plain
    assert gba.gba_aggregate_apply_sparse_workspace_size(n, 3, 32, 1000, "adam") >= plain + n * 32 * 4
    assert gba.gba_aggregate_apply_sparse_workspace_size(n, 3, 64, 1000, "adagrad") >= \
        gba.gba_aggregate_sparse_workspace_size(n, 3, 64, 1000) + n * 64 * 4
