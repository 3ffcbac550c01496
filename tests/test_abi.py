"""The C ABI without a GPU: the built library loads, exports every function
include/qe.h declares (and no undeclared qe_ symbol), and its host-only
helpers (status strings, version, workspace and packing sizes) answer as
documented, and host-detectable argument errors are reported before any
device work.  No call here launches a kernel or touches a device."""
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
    texts = [L.qe_status_string(c).decode() for c in range(9)]
    assert texts[0] == "ok"
    assert len(set(texts)) == 9 and all(texts)
    assert L.qe_status_string(99).decode() == "unknown status"
    assert L.qe_version() == 1


def test_workspace_sizes(lib):
    """Host arithmetic only.  The Gram's size pins its token-split choice:
    4096 channels x 262144 tokens -> 15 splits of the 528 upper-triangle
    128 x 128 tiles (64 KiB each) after the 256-byte status word; at 59392
    channels the partials would not fit, so Sigma is written directly.  Then
    the channel exponents of the fp16 split (p ints) and the token-major
    pre-pass partials (slices x p floats: about 2048 workgroups of 1024
    channels, at least 256 tokens a slice; 512 slices at p = 4096 and 262144
    tokens, 128 at 32768 tokens, 35 at p = 59392)."""
    L, _ = lib
    for f in ("qe_gram_workspace_size", "qe_cd_workspace_size", "qe_objective_workspace_size",
              "qe_lambda_workspace_size", "qe_outlier_workspace_size", "qe_topk_workspace_size",
              "qe_topk_columns_workspace_size"):
        getattr(L, f).restype = ctypes.c_size_t
    L.qe_gram_workspace_size.argtypes = [ctypes.c_int64, ctypes.c_int64]
    assert L.qe_gram_workspace_size(4096, 262144) == 256 + 15 * 528 * 65536 + 4096 * 4 + 512 * 4096 * 4
    assert L.qe_gram_workspace_size(59392, 32768) == 256 + 59392 * 4 + 35 * 59392 * 4
    # a 32768-token chunk at 4096 channels: 13 splits of 2528 tokens fill the 256 CUs
    assert (L.qe_gram_workspace_size(4096, 32768) ==
            256 + 13 * 528 * 65536 + 4096 * 4 + 128 * 4096 * 4)
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


def test_binding_constants_match_the_header():
    """Every object-like QE_ macro of qe.h (status codes, layouts, flags,
    sizes) has the same value in the binding and is re-exported by the
    package."""
    import paper_2309_01885_amd as P
    import paper_2309_01885_amd.qe as Q
    text = re.sub(r"/\*.*?\*/", " ", open(HEADER).read(), flags=re.S)
    macros = re.findall(r"^#define[ \t]+(QE_[A-Z0-9_]+)[ \t]+(.+?)[ \t]*$", text, flags=re.M)
    assert {"QE_OK", "QE_OBJ_IN", "QE_NOALLOC_SCRATCH_BYTES"} <= {n for n, _ in macros}
    for name, raw in macros:
        # integer literals (u suffix dropped) and shifts of them
        expr = re.sub(r"\b(0x[0-9a-fA-F]+|[0-9]+)u\b", r"\1", raw)
        assert re.fullmatch(r"[0-9a-fA-Fx()<< ]+", expr), (name, raw)
        value = eval(expr)
        assert getattr(Q, name) == value, name
        assert getattr(P, name) == value, name


# ------------------------------------------------------------------ argument errors
# Host-detectable argument errors return before any HIP call (qe.h: errors),
# so they are checked here without a GPU.  Pointers are dummies: none is
# dereferenced on these paths.
QE_ERR_ARG, QE_ERR_WORKSPACE = 1, 4
DUMMY = ctypes.c_void_p(4096)
NULL = ctypes.c_void_p(0)


def _gram(L, X=DUMMY, p=64, n=64, layout=0, S=DUMMY, damp=0.0, ws=DUMMY, ws_bytes=1 << 40):
    f = L.qe_gram
    f.restype = ctypes.c_int
    f.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64, ctypes.c_int, ctypes.c_void_p,
                  ctypes.c_int, ctypes.c_float, ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p]
    return f(X, p, n, layout, S, 0, damp, ws, ws_bytes, NULL)


def test_gram_argument_errors(lib):
    L, _ = lib
    assert _gram(L, X=NULL) == QE_ERR_ARG
    assert _gram(L, S=NULL) == QE_ERR_ARG
    assert _gram(L, p=0) == QE_ERR_ARG            # empty input
    assert _gram(L, n=0) == QE_ERR_ARG
    assert _gram(L, layout=2) == QE_ERR_ARG
    assert _gram(L, layout=0x100 | 0x200) == QE_ERR_ARG   # QE_GRAM_FP32 with QE_GRAM_BF16X3
    assert _gram(L, layout=0x400) == QE_ERR_ARG           # no such flag
    assert _gram(L, layout=0x200 | 1, ws=NULL) == QE_ERR_WORKSPACE   # QE_GRAM_BF16X3 is accepted
    assert _gram(L, damp=-1.0) == QE_ERR_ARG
    assert _gram(L, damp=float("nan")) == QE_ERR_ARG
    assert _gram(L, ws=NULL) == QE_ERR_WORKSPACE
    assert _gram(L, ws_bytes=16) == QE_ERR_WORKSPACE


def _cd(L, q=64, p=64, bits=4, sweeps=1, block=0, flags=0, ws=DUMMY, ws_bytes=1 << 40, W=DUMMY,
        obj=NULL):
    f = L.qe_cd_sweep
    f.restype = ctypes.c_int
    f.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64, ctypes.c_int,
                  ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                  ctypes.c_void_p, ctypes.c_int, ctypes.c_int, ctypes.c_uint32, ctypes.c_void_p,
                  ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p]
    return f(W, DUMMY, q, p, bits, DUMMY, DUMMY, DUMMY, DUMMY, DUMMY, sweeps, block, flags, obj,
             ws, ws_bytes, NULL)


def test_cd_sweep_argument_errors(lib):
    L, _ = lib
    assert _cd(L, W=NULL) == QE_ERR_ARG
    assert _cd(L, q=0) == QE_ERR_ARG              # empty input
    assert _cd(L, p=0) == QE_ERR_ARG
    assert _cd(L, bits=0) == QE_ERR_ARG           # bits outside [1, 8]
    assert _cd(L, bits=9) == QE_ERR_ARG
    assert _cd(L, block=48) == QE_ERR_ARG         # block widths 16, 32, 64, 128 (0 = default)
    assert _cd(L, sweeps=-1) == QE_ERR_ARG
    assert _cd(L, flags=0x10) == QE_ERR_ARG       # QE_OUTLIER_COLUMNS belongs to the outlier call
    assert _cd(L, flags=0x20000) == QE_ERR_ARG    # no such flag
    assert _cd(L, flags=0x10000, ws=NULL) == QE_ERR_WORKSPACE   # QE_CD_DENSE is accepted
    assert _cd(L, flags=0x40, ws=NULL) == QE_ERR_WORKSPACE   # QE_DEBUG_CHECKS is accepted
    # QE_OBJ_IN reads obj[0]: it needs obj, and not with QE_INIT_FROM_W
    assert _cd(L, flags=0x80) == QE_ERR_ARG
    assert _cd(L, flags=0x80 | 0x1, obj=DUMMY) == QE_ERR_ARG
    assert _cd(L, flags=0x80 | 0x2, obj=DUMMY, ws=NULL) == QE_ERR_WORKSPACE
    assert _cd(L, ws=NULL) == QE_ERR_WORKSPACE
    assert _cd(L, ws_bytes=1024) == QE_ERR_WORKSPACE


def test_cd_sweep_noalloc_argument_errors(lib):
    """The allocation-free variant checks its arguments like qe_cd_sweep and
    rejects sizes whose scratch exceeds the fixed array (64 MiB) before any
    HIP call."""
    L, _ = lib
    f = L.qe_cd_sweep_noalloc
    f.restype = ctypes.c_int
    f.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64, ctypes.c_int64, ctypes.c_int,
                  ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p, ctypes.c_void_p,
                  ctypes.c_void_p, ctypes.c_int, ctypes.c_int, ctypes.c_uint32, ctypes.c_void_p,
                  ctypes.c_void_p, ctypes.c_void_p]

    def call(W=DUMMY, q=64, p=64, bits=4, block=0, flags=0, obj=NULL):
        return f(W, DUMMY, q, p, bits, DUMMY, DUMMY, DUMMY, DUMMY, DUMMY, 1, block, flags, obj,
                 NULL, NULL)
    assert call(W=NULL) == QE_ERR_ARG
    assert call(flags=0x80) == QE_ERR_ARG              # QE_OBJ_IN without obj
    assert call(flags=0x81, obj=DUMMY) == QE_ERR_ARG   # QE_OBJ_IN with QE_INIT_FROM_W
    assert call(bits=9) == QE_ERR_ARG
    assert call(block=48) == QE_ERR_ARG
    L.qe_cd_workspace_size.restype = ctypes.c_size_t
    L.qe_cd_workspace_size.argtypes = [ctypes.c_int64, ctypes.c_int64, ctypes.c_int]
    assert L.qe_cd_workspace_size(40000, 4096, 0) > (64 << 20)
    assert call(q=40000, p=4096) == 7                  # QE_ERR_TOO_LARGE
    assert L.qe_cd_workspace_size(14848, 59392, 0) <= (64 << 20)   # the largest workload fits


def test_lambda_and_objective_argument_errors(lib):
    L, _ = lib
    f = L.qe_lambda_max
    f.restype = ctypes.c_int
    f.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_float, ctypes.c_void_p,
                  ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p]
    out = ctypes.c_float(0.0)
    assert f(DUMMY, 64, 0, 1e-7, ctypes.byref(out), DUMMY, 1 << 40, NULL) == QE_ERR_ARG
    assert f(DUMMY, 0, 10, 1e-7, ctypes.byref(out), DUMMY, 1 << 40, NULL) == QE_ERR_ARG
    assert f(DUMMY, 64, 10, float("nan"), ctypes.byref(out), DUMMY, 1 << 40, NULL) == QE_ERR_ARG
    assert f(DUMMY, 64, 10, 1e-7, ctypes.byref(out), DUMMY, 8, NULL) == QE_ERR_WORKSPACE
    g = L.qe_objective
    g.restype = ctypes.c_int
    g.argtypes = [ctypes.c_void_p] * 4 + [ctypes.c_int64, ctypes.c_int64, ctypes.c_void_p,
                                          ctypes.c_void_p, ctypes.c_size_t, ctypes.c_void_p]
    assert g(DUMMY, NULL, NULL, DUMMY, 8, 8, DUMMY, DUMMY, 1 << 40, NULL) == QE_ERR_ARG
    assert g(DUMMY, DUMMY, NULL, DUMMY, 0, 8, DUMMY, DUMMY, 1 << 40, NULL) == QE_ERR_ARG
    assert g(DUMMY, DUMMY, NULL, DUMMY, 8, 8, DUMMY, DUMMY, 8, NULL) == QE_ERR_WORKSPACE


def test_peak_library_exports_and_argument_errors():
    """libqe_peak.so (peak checks) loads and rejects bad arguments before any launch."""
    from paper_2309_01885_amd import peaks
    L = peaks.load()
    assert L.qpk_mfma_bf16(None, 512, 10, None) == 1
    assert L.qpk_mfma_f16(DUMMY, 512, 0, None) == 1
    assert L.qpk_mfma_f32(DUMMY, 0, 10, None) == 1
    assert L.qpk_clock(DUMMY, None, 512, 10, None) == 1
    assert L.qpk_copy(DUMMY, ctypes.c_void_p(4100), 16, 64, 0, None) == 1    # misaligned
    assert L.qpk_copy(DUMMY, DUMMY, 0, 64, 1, None) == 1
