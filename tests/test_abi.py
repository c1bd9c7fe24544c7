"""The C ABI: the library loads, exports every declared entry point, answers
size queries and rejects bad arguments on the host before any launch."""
import ctypes
import os
import shutil
import subprocess
import sys

import pytest

from helpers import header_functions, ROOT

LIB = os.path.join(ROOT, "paper_2303_07030_amd", "libnsd.so")


@pytest.fixture(scope="module")
def nsd():
    if not os.path.exists(LIB):
        pytest.fail("libnsd.so is not built; run __graft_entry__.build()")
    from paper_2303_07030_amd import nsd as m
    return m


def test_header_declares_entry_points():
    names = header_functions()
    assert "nsd_loss_frob_spmm" in names and "nsd_csr_to_csc" in names
    assert len(names) >= 15


def test_every_declared_symbol_is_exported(nsd):
    lib = ctypes.CDLL(LIB)
    missing = [n for n in header_functions() if not hasattr(lib, n)]
    assert not missing, f"declared but not exported: {missing}"


def test_binding_covers_every_declared_symbol(nsd):
    assert sorted(nsd.EXPORTED) == header_functions()
    for n in header_functions():
        assert callable(getattr(nsd, n)), n


def test_exports_are_c_symbols():
    out = subprocess.run(["nm", "-D", "--defined-only", LIB], capture_output=True, text=True).stdout
    syms = {line.split()[-1] for line in out.splitlines() if line.strip()}
    for n in header_functions():
        assert n in syms, f"{n} missing or mangled"


def test_status_strings_and_version(nsd):
    assert nsd.nsd_status_string(0) == "NSD_OK"
    assert nsd.nsd_status_string(5) == "NSD_ERR_WORKSPACE"
    assert nsd.nsd_status_string(99) == "NSD_ERR_UNKNOWN"
    assert nsd.nsd_version() >= 100


def _desc(nsd, nrows=4, ncols=4, nnz=3, ptr=0x1000, nitems=1):
    d = nsd.nsd_csr(nrows, ncols, nnz, ptr, ptr, ptr, ptr)
    d.plan = nsd.nsd_plan(16, nitems, 0, 0, 0, 0, ptr, 0, 0, 0, 0, 0)
    return d


def test_workspace_queries(nsd):
    # descriptors with plans of 100 and 10,000 items: sizes only, nothing is read
    small = nsd.nsd_workspace_size(_desc(nsd, 1000, 1000, 5000, nitems=100), None, 64)
    big = nsd.nsd_workspace_size(_desc(nsd, 1000, 1000, 5000, nitems=10_000), None, 64)
    assert 0 < small < big and big % 256 == 0
    assert nsd.nsd_build_workspace_size(0, 1) > 0
    with pytest.raises(nsd.NsdError) as e:
        nsd.nsd_workspace_size(_desc(nsd), None, 0)
    assert e.value.status == nsd.NSD_ERR_INVALID_ARG
    mi, ml, mc, wb = nsd.nsd_plan_bounds(100_000, 1_000_000, 32)
    assert mi >= 100_000 and ml >= 1 and mc >= 2 * 1_000_000 // 32 and wb > 0
    assert 16 <= nsd.nsd_plan_item_len(1_000_000, 64) <= 256
    # shorter items only where 16-entry ones leave SIMDs without a wave
    assert nsd.nsd_plan_item_len(10_000, 1) == 2
    assert nsd.nsd_plan_item_len(0, 64) == 2
    for k in (1, 12, 64, 300):
        ls = [nsd.nsd_plan_item_len(n, k) for n in (0, 10**3, 10**4, 10**5, 10**6, 10**7, 10**8)]
        assert ls == sorted(ls) and 2 <= ls[0] and ls[-1] <= 256, (k, ls)
    with pytest.raises(nsd.NsdError) as e:
        nsd.nsd_plan_bounds(10, 2**30, 16)
    assert e.value.status == nsd.NSD_ERR_TOO_LARGE


def test_host_argument_errors_before_launch(nsd):
    # every call below must be rejected on the host: no pointer is ever read
    with pytest.raises(nsd.NsdError) as e:
        nsd._check(nsd._lib.nsd_spmm(None, None, 64, None, None, 0, None), "nsd_spmm")
    assert e.value.status == nsd.NSD_ERR_INVALID_ARG
    A = _desc(nsd)
    with pytest.raises(nsd.NsdError) as e:
        nsd.nsd_spmm(A, 0x1000, 0, 0x1000, None)            # k < 1
    assert e.value.status == nsd.NSD_ERR_INVALID_ARG
    with pytest.raises(nsd.NsdError) as e:
        nsd.nsd_spmm(A, 0x1000, 8, 0x1000, None)            # no workspace
    assert e.value.status == nsd.NSD_ERR_WORKSPACE
    noplan = nsd.nsd_csr(4, 4, 3, 0x1000, 0x1000, 0x1000, 0x1000)
    with pytest.raises(nsd.NsdError) as e:
        nsd.nsd_spmm(noplan, 0x1000, 8, 0x1000, None)       # plan never built
    assert e.value.status == nsd.NSD_ERR_INVALID_ARG and "plan" in str(e.value)
    bad = nsd.nsd_csr(-1, 4, 3, 0x1000, 0x1000, 0x1000, 0x1000)
    with pytest.raises(nsd.NsdError) as e:
        nsd.nsd_sddmm(bad, None, 0x1000, 4, 1.0, 0x1000)
    assert e.value.status == nsd.NSD_ERR_INVALID_ARG
    At = nsd.nsd_csc(4, 5, 3, 0x1000, 0x1000, 0x1000, 0x1000)  # shape mismatch
    with pytest.raises(nsd.NsdError) as e:
        nsd.nsd_spmm_t(A, At, None, 1, 1.0, 0x1000, None)
    assert e.value.status == nsd.NSD_ERR_INVALID_ARG
    with pytest.raises(nsd.NsdError) as e:
        nsd.nsd_coo_to_csr(4, 4, 3, 0x1000, 0x1000, 0x1000, 7, 0x1000, 0x1000, 0x1000, 0x1000,
                           0x1000, None)                      # unknown policy
    assert e.value.status == nsd.NSD_ERR_INVALID_ARG
    with pytest.raises(nsd.NsdError) as e:
        nsd.nsd_coo_mode_index(3, 0, 0x1000, 0x1000, 0x1000, 0x1000, None)   # dim < 1
    assert e.value.status == nsd.NSD_ERR_INVALID_ARG
    assert "dim" in nsd.nsd_last_error()
    with pytest.raises(nsd.NsdError) as e:
        nsd.nsd_diag_keys(A, 1.0, None)                     # no output for 3 entries
    assert e.value.status == nsd.NSD_ERR_INVALID_ARG
    T = nsd.nsd_ttv_plan()
    with pytest.raises(nsd.NsdError) as e:
        nsd.nsd_ttm_workspace_size(T, 8)                    # order 0: not a built plan
    assert e.value.status == nsd.NSD_ERR_INVALID_ARG
    T.order, T.mode = 3, 2
    T.dims[:3] = (4, 4, 4)
    with pytest.raises(nsd.NsdError) as e:
        nsd.nsd_ttm_workspace_size(T, 0)                    # R < 1
    assert e.value.status == nsd.NSD_ERR_INVALID_ARG
    with pytest.raises(nsd.NsdError) as e:
        nsd.nsd_ttm(T, None, None, 8, None, None)           # empty plan, no workspace
    assert e.value.status == nsd.NSD_ERR_WORKSPACE
    T.nnz = 5
    with pytest.raises(nsd.NsdError) as e:
        nsd.nsd_ttm_vjp(T, 0x1000, 0x1000, 8, 0x1000, 0x1000, 0x1000, None)  # plan not built
    assert e.value.status == nsd.NSD_ERR_INVALID_ARG
    dims = (4, 4, 4, 4)
    for order, mode in ((2, 0), (7, 0), (4, 4), (4, -1)):
        with pytest.raises(nsd.NsdError) as e:              # order or mode out of range
            nsd.nsd_ttv_build(order, dims[:max(min(order, 4), 1)] * 2, 3, [0x1000] * 4, mode,
                              [0x1000] * 3, 0x1000, 0x1000, 0x1000, 0x1000, 0x1000, 0x1000,
                              0x1000, 0x1000, None)
        assert e.value.status == nsd.NSD_ERR_INVALID_ARG


def test_binding_fails_loudly_without_library(tmp_path):
    # a copy of the binding next to no library must refuse to import
    pkg = tmp_path / "paper_2303_07030_amd"
    pkg.mkdir()
    shutil.copy(os.path.join(ROOT, "paper_2303_07030_amd", "nsd.py"), pkg / "nsd.py")
    (pkg / "__init__.py").write_text("")
    r = subprocess.run([sys.executable, "-c", "import paper_2303_07030_amd.nsd"], cwd=tmp_path,
                       capture_output=True, text=True)
    assert r.returncode != 0 and "libnsd.so is not built" in r.stderr


def test_probe_accepts_every_kernel_id():
    """Every kernel id the header declares is known to the binding and is
    accepted by nsd_probe_set (fake handles: no kernel runs, so they are
    never recorded), and an unknown one is refused."""
    import re
    from paper_2303_07030_amd import nsd
    text = open(os.path.join(ROOT, "include", "nsd.h")).read()
    ids = {m.group(1).lower(): int(m.group(2))
           for m in re.finditer(r"NSD_KERNEL_(\w+)\s*=\s*(\d+)", text) if m.group(1) != "NONE"}
    assert ids == nsd.KERNEL_IDS
    for kid in ids.values():
        nsd.nsd_probe_set(kid, [1], [1])
        assert nsd.nsd_probe_count() == 0
        nsd.nsd_probe_clear()
    with pytest.raises(nsd.NsdError):
        nsd.nsd_probe_set(max(ids.values()) + 1, [1], [1])
