"""Host-side checks of the C-ABI library that need no GPU: it loads and
exports every entry point include/routepack.h declares, and argument errors
are reported before any device work."""
import ctypes as C
import os
import re

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared(header="routepack.h"):
    src = open(os.path.join(ROOT, "include", header)).read()
    return sorted(set(re.findall(r"^(?:int|const char \*)\s*(routepack_\w+)\s*\(", src, re.M)))


def test_header_declares_the_boundary():
    assert _declared() == sorted(["routepack_aggregate_demand", "routepack_aggregate_demand_noalloc",
                                  "routepack_place_experts",
                                  "routepack_pack_rows", "routepack_anneal",
                                  "routepack_eval_objective", "routepack_select_population",
                                  "routepack_row_lower_bound", "routepack_fixed_bin_search", "routepack_project_demand",
                                  "routepack_strerror"])


def test_library_exports_every_declared_symbol():
    import paper_2608_12146_amd as rp
    lib = rp.load_library()
    headers = sorted(f for f in os.listdir(os.path.join(ROOT, "include")) if f.endswith(".h"))
    assert headers == ["routepack.h", "routepack_probe.h"]
    for name in _declared("routepack.h"):
        assert hasattr(lib, name), name
    # the LDS probe (a measurement aid) lives in its own library only
    probe = rp.load_probe_library()
    assert _declared("routepack_probe.h") == list(rp.PROBE_EXPORTS)
    for name in rp.PROBE_EXPORTS:
        assert hasattr(probe, name), name
        assert not hasattr(lib, name), name
    assert lib.routepack_strerror(-5) == b"fixed-point score bound exceeds 2^53"


def test_lds_probe_rejects_bad_arguments_without_device_work():
    import paper_2608_12146_amd as rp
    lib = rp.load_probe_library()
    ms, nb = C.c_double(0.0), C.c_int64(0)
    assert lib.routepack_probe_lds_read(0, 1, C.c_void_p(16), C.byref(ms), C.byref(nb), None) == -1
    assert lib.routepack_probe_lds_read(1, 0, C.c_void_p(16), C.byref(ms), C.byref(nb), None) == -1
    assert lib.routepack_probe_lds_read(1, 1, None, C.byref(ms), C.byref(nb), None) == -1
    assert lib.routepack_probe_lds_read(1 << 30, 1 << 30, C.c_void_p(16), C.byref(ms), C.byref(nb), None) == -1


def test_invalid_problems_rejected_without_device_work():
    import paper_2608_12146_amd as rp
    lib = rp.load_library()
    # E % P != 0 and a shard with no slot: rejected during validation.
    bad = rp.Problem(8, 2, 6, 2, 4, 2, 1, [0, 0], 64, [4096], [1])
    assert lib.routepack_eval_objective(bad.ref, None, None, 1, 0, None, None, None, None, None,
                                        None, None) == -1
    bad2 = rp.Problem(8, 2, 8, 2, 4, 2, 2, [0, 0], 64, [4096], [1])
    assert lib.routepack_anneal(bad2.ref, None, None, 1, 1, None, None, None, None, None, None,
                                None, None) == -1
    assert lib.routepack_place_experts(bad.ref, None, None, None, None, None, None) == -1
    assert lib.routepack_aggregate_demand(None, None, None, None) == -1


def test_noalloc_aggregation_rejects_oversized_shapes_without_device_work():
    """routepack_aggregate_demand_noalloc refuses L E > 2^20 (one band of
    partials would not fit its fixed array) before any HIP call."""
    import paper_2608_12146_amd as rp
    lib = rp.load_library()
    big = rp.Problem(1, 1, (1 << 20) + 1, 1, 1, 1, 1, [0], 64, [4096], [1])
    assert lib.routepack_aggregate_demand_noalloc(big.ref, C.c_void_p(16), C.c_void_p(16), None) == -8
    assert lib.routepack_aggregate_demand_noalloc(None, None, None, None) == -1
