"""The C ABI without a GPU: the built library loads, exports every function
include/qe.h declares (and no undeclared qe_ symbol), and its host-only
helpers (status strings, version, workspace and packing sizes) answer as
documented.  No call here launches a kernel or touches a device."""
import ctypes
import os
import re
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "qe.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
    text = re.sub(r"//[^\n]*", " ", text)
    names = re.findall(r"^[ \t]*(?:const[ \t]+)?[A-Za-z_][\w]*[ \t\*]+(qe_[a-z0-9_]+)[ \t]*\(",
                       text, flags=re.M)
    return sorted(set(names))


@pytest.fixture(scope="module")
def lib():
    import paper_2309_01885_amd.qe as Q
    assert os.path.exists(Q.LIB_PATH), "libqe.so not built (run __graft_entry__.build())"
    return ctypes.CDLL(Q.LIB_PATH), Q.LIB_PATH


def test_header_declares_the_entry_points():
    names = declared_functions()
    for must in ("qe_gram", "qe_cd_sweep", "qe_cd_outlier_sweep", "qe_objective",
                 "qe_grid_minmax", "qe_lambda_max", "qe_gram_workspace_size",
                 "qe_cd_workspace_size", "qe_status_string", "qe_sync_status"):
        assert must in names
    assert len(names) >= 20


def test_every_declared_function_is_exported(lib):
    L, _ = lib
    missing = [n for n in declared_functions() if not hasattr(L, n)]
    assert not missing, missing


@pytest.mark.skipif(shutil.which("nm") is None, reason="nm not installed")
def test_no_undeclared_exports(lib):
    _, path = lib
    out = subprocess.run(["nm", "-D", "--defined-only", path], capture_output=True, text=True,
                         check=True).stdout
    exported = sorted({ln.split()[-1] for ln in out.splitlines()
                       if ln.split() and ln.split()[-1].startswith("qe_")
                       and ln.split()[-2] in ("T", "t", "W")})
    assert exported == declared_functions()


def test_status_strings_and_version(lib):
    L, _ = lib
    L.qe_status_string.restype = ctypes.c_char_p
    L.qe_status_string.argtypes = [ctypes.c_int]
    texts = [L.qe_status_string(c).decode() for c in range(7)]
    assert texts[0] == "ok"
    assert len(set(texts)) == 7 and all(texts)
    assert L.qe_status_string(99).decode() == "unknown status"
    assert L.qe_version() == 1


def test_workspace_sizes(lib):
    """Host arithmetic only.  The Gram's size pins its token-split choice:
    4096 channels x 262144 tokens -> 15 splits of the 528 upper-triangle
    128 x 128 tiles (64 KiB each) after the 256-byte status word; at 59392
    channels the partials would not fit, so Sigma is written directly."""
    L, _ = lib
    for f in ("qe_gram_workspace_size", "qe_cd_workspace_size", "qe_objective_workspace_size",
              "qe_lambda_workspace_size", "qe_outlier_workspace_size", "qe_topk_workspace_size",
              "qe_topk_columns_workspace_size"):
        getattr(L, f).restype = ctypes.c_size_t
    L.qe_gram_workspace_size.argtypes = [ctypes.c_int64, ctypes.c_int64]
    assert L.qe_gram_workspace_size(4096, 262144) == 256 + 15 * 528 * 65536
    assert L.qe_gram_workspace_size(59392, 32768) == 256
    assert L.qe_gram_workspace_size(0, 10) == 256
    L.qe_cd_workspace_size.argtypes = [ctypes.c_int64, ctypes.c_int64, ctypes.c_int]
    c2 = L.qe_cd_workspace_size(4096, 4096, 0)
    assert c2 >= 2 * 4096 * 256 * 4                    # the two delta buffers
    assert L.qe_cd_workspace_size(4096, 4096, 128) == c2
    assert L.qe_cd_workspace_size(0, 4096, 0) == 0       # bad dimensions
    assert L.qe_cd_workspace_size(4096, 4096, 7) == 0    # bad block width
    L.qe_outlier_workspace_size.argtypes = [ctypes.c_int64, ctypes.c_int64, ctypes.c_int,
                                            ctypes.c_int64]
    assert L.qe_outlier_workspace_size(4096, 4096, 0, 167772) > c2
    L.qe_objective_workspace_size.argtypes = [ctypes.c_int64, ctypes.c_int64]
    assert L.qe_objective_workspace_size(4096, 4096) >= 256
    L.qe_lambda_workspace_size.argtypes = [ctypes.c_int64]
    assert L.qe_lambda_workspace_size(4096) >= 256


@pytest.mark.parametrize("bits", [1, 2, 3, 4, 8])
def test_packed_row_bytes(lib, bits):
    L, _ = lib
    L.qe_packed_row_bytes.restype = ctypes.c_int64
    L.qe_packed_row_bytes.argtypes = [ctypes.c_int64, ctypes.c_int]
    for p in (1, 7, 512, 4096, 4097):
        assert L.qe_packed_row_bytes(p, bits) == (p * bits + 7) // 8
    assert L.qe_packed_row_bytes(16, 0) == 0
    assert L.qe_packed_row_bytes(16, 9) == 0


def test_binding_names_follow_the_abi():
    """Each compute entry point qe_X has the binding function X."""
    import paper_2309_01885_amd.qe as Q
    helpers = {"qe_version", "qe_packed_row_bytes"}
    for n in declared_functions():
        if n.endswith("_workspace_size") or n in helpers:
            continue
        assert callable(getattr(Q, n[len("qe_"):], None)), n
