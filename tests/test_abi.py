"""Host-only checks of the C ABI boundary (no GPU needed, no compute calls).

* libpardnn.so (built for gfx950 by hipcc) loads and exports every function
  that include/pardnn.h declares, and nothing is left undeclared;
* status strings and the no-GPU error path (E_DEVICE) behave as documented;
* the Python binding refuses to run without the library (no CPU fallback);
* the oracle and the HIP library share no source file, header or include.
"""
import glob
import os
import re
import subprocess

import pytest
import torch

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "pardnn.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(pardnn_[a-z_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def lib():
    import paper_2008_08636_amd as P
    from paper_2008_08636_amd import build
    if not os.path.exists(P.LIB_PATH):
        build.build()
    return P.load_library()


def test_header_declares_the_boundary():
    names = declared_functions()
    for required in ["pardnn_graph_create", "pardnn_graph_destroy", "pardnn_levelize",
                     "pardnn_tb_levels", "pardnn_critical_path", "pardnn_label_memory",
                     "pardnn_apply_moves", "pardnn_build_placements", "pardnn_evaluate_batch",
                     "pardnn_tb_levels_batch", "pardnn_status_string", "pardnn_last_error"]:
        assert required in names


def test_library_exports_every_declared_symbol(lib):
    import paper_2008_08636_amd as P
    out = subprocess.run(["nm", "-D", "--defined-only", P.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = set(re.findall(r"\bT (pardnn_[a-z_]+)$", out, flags=re.M))
    declared = set(declared_functions())
    assert declared <= exported, declared - exported
    assert exported <= declared, exported - declared
    for name in declared:
        getattr(lib, name)


def test_library_targets_gfx950_only():
    import paper_2008_08636_amd as P
    blob = open(P.LIB_PATH, "rb").read()
    # the offload bundle names one target per code object; host code may
    # still hold other architecture names (a library's arch dispatch tables)
    targets = set(re.findall(rb"amdgcn-amd-amdhsa--(gfx[0-9a-f]+)", blob))
    assert targets == {b"gfx950"}, targets


def test_status_strings(lib):
    import paper_2008_08636_amd as P
    assert P.pardnn_status_string(0) == "ok"
    assert "cycle" in P.pardnn_status_string(P.E_CYCLE)
    assert P.pardnn_status_string(123) == "unknown status"


def test_null_arguments_rejected_on_host(lib):
    import ctypes
    h = ctypes.c_void_p()
    # n_edges > 0 with null edge arrays: rejected before any device call
    assert lib.pardnn_graph_create(3, 2, None, None, None, None, None, None, ctypes.byref(h)) == -1
    assert lib.pardnn_graph_create(-1, 0, None, None, None, None, None, None, ctypes.byref(h)) == -1
    assert lib.pardnn_graph_create(0, 0, None, None, None, None, None, None, None) == -1
    # size limits: 2^26 nodes, 2^27 edges (checked before anything is read)
    assert lib.pardnn_graph_create((1 << 26) + 1, 0, None, None, None, None, None, None,
                                   ctypes.byref(h)) == -1
    assert lib.pardnn_graph_create(4, (1 << 27) + 1, None, None, None, None, None, None,
                                   ctypes.byref(h)) == -1
    assert b"2^26" in lib.pardnn_last_error()
    assert lib.pardnn_tb_levels(None, None, None, None, None) == -1
    assert b"null" in lib.pardnn_last_error()


@pytest.mark.skipif(torch.cuda.is_available(), reason="checks the no-GPU path")
def test_no_device_reports_e_device(lib):
    import ctypes
    h = ctypes.c_void_p()
    st = lib.pardnn_graph_create(0, 0, None, None, None, None, None, None, ctypes.byref(h))
    assert st == -5 and not h.value


def test_fault_alloc_hook_reports_e_nomem(lib, monkeypatch):
    """PARDNN_FAULT_ALLOC=n fails the n-th allocation attempt as out of
    memory; the handle is the first allocation of pardnn_graph_create and
    needs no device, so n = 1 gives E_NOMEM here as on a GPU."""
    import ctypes
    h = ctypes.c_void_p()
    monkeypatch.setenv("PARDNN_FAULT_ALLOC", "1")
    assert lib.pardnn_graph_create(0, 0, None, None, None, None, None, None,
                                   ctypes.byref(h)) == -4
    assert not h.value and b"host allocation" in lib.pardnn_last_error()
    # one failure per value of the variable: the next attempt goes through
    st = lib.pardnn_graph_create(0, 0, None, None, None, None, None, None, ctypes.byref(h))
    assert st in (0, -5)
    if st == 0:
        assert lib.pardnn_graph_destroy(h) == 0
    # a new value restarts the count; 0 and empty never fail
    monkeypatch.setenv("PARDNN_FAULT_ALLOC", "01")
    assert lib.pardnn_graph_create(0, 0, None, None, None, None, None, None,
                                   ctypes.byref(h)) == -4
    for v in ("0", ""):
        monkeypatch.setenv("PARDNN_FAULT_ALLOC", v)
        st = lib.pardnn_graph_create(0, 0, None, None, None, None, None, None, ctypes.byref(h))
        assert st in (0, -5)
        if st == 0:
            assert lib.pardnn_graph_destroy(h) == 0
    # argument errors come before any allocation
    monkeypatch.setenv("PARDNN_FAULT_ALLOC", "1")
    assert lib.pardnn_graph_create(-1, 0, None, None, None, None, None, None,
                                   ctypes.byref(h)) == -1


def test_binding_has_no_fallback(monkeypatch, tmp_path):
    import paper_2008_08636_amd as P
    monkeypatch.setattr(P, "_lib", None)
    with pytest.raises(RuntimeError, match="not built"):
        P.load_library(str(tmp_path / "missing.so"))


def test_oracle_and_library_share_nothing():
    csrc = glob.glob(os.path.join(ROOT, "paper_2008_08636_amd", "csrc", "*"))
    for f in csrc:
        text = open(f).read()
        assert "oracle" not in text.lower(), f
    for f in glob.glob(os.path.join(ROOT, "oracle", "*.[ch]")):
        text = open(f).read()
        assert "pardnn.h" not in text and "csrc" not in text, f
    pkg = open(os.path.join(ROOT, "paper_2008_08636_amd", "__init__.py")).read()
    assert "import oracle" not in pkg and "from oracle" not in pkg
