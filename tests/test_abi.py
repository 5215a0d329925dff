"""C-ABI contract checks that need no GPU: the library loads, exports every
declared entry point, and rejects bad arguments before touching a device."""
import ctypes
import os
import re

import pytest

from conftest import ROOT, gpu_available

HEADER = os.path.join(ROOT, "include", "dualgcn.h")


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(dualgcn_[a-z_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def dg():
    import paper_2609_01983_amd as dg
    return dg


def test_every_declared_symbol_is_exported(dg):
    names = _declared()
    assert len(names) >= 10
    for name in names:
        assert hasattr(dg.lib(), name), name


def test_status_strings(dg):
    for code in range(-6, 1):
        assert dg.status_str(code) and dg.status_str(code) != "unknown status"
    assert dg.status_str(42) == "unknown status"


def _csr(dg, n=4, nnz=4, rowptr=1, col=1, val=1):
    return dg.Csr(n, nnz, rowptr, col, val)


def test_partition_argument_checks(dg):
    L = dg.lib()
    out = ctypes.c_void_p(123)
    assert L.dualgcn_partition(None, 0, 4, 4, None, None, ctypes.byref(out)) == dg.ERR_INVALID_ARG
    assert out.value is None                         # *out cleared on error
    c = _csr(dg)
    assert L.dualgcn_partition(ctypes.byref(c), 0, 4, 4, None, None, None) == dg.ERR_INVALID_ARG
    assert L.dualgcn_partition(ctypes.byref(c), 0, 0, 4, None, None, ctypes.byref(out)) == dg.ERR_INVALID_ARG
    assert L.dualgcn_partition(ctypes.byref(c), 0, 4, 0, None, None, ctypes.byref(out)) == dg.ERR_INVALID_ARG
    assert L.dualgcn_partition(ctypes.byref(c), 0, 4, 256, None, None, ctypes.byref(out)) == dg.ERR_UNSUPPORTED
    # S_v <= k (d + 1) must fit 32 bits
    assert L.dualgcn_partition(ctypes.byref(c), 0, 1 << 28, 15, None, None, ctypes.byref(out)) == dg.ERR_UNSUPPORTED
    assert L.dualgcn_partition(ctypes.byref(c), 0, (1 << 28) - 1, 15, None, None,
                               ctypes.byref(out)) == dg.ERR_NO_DEVICE
    big = _csr(dg, nnz=1 << 31)
    assert L.dualgcn_partition(ctypes.byref(big), 0, 4, 4, None, None, ctypes.byref(out)) == dg.ERR_UNSUPPORTED
    for bad in [_csr(dg, n=0), _csr(dg, nnz=-1), _csr(dg, rowptr=0), _csr(dg, col=0)]:
        assert L.dualgcn_partition(ctypes.byref(bad), 0, 4, 4, None, None, ctypes.byref(out)) == dg.ERR_INVALID_ARG
    for th in [dg.Thresholds(1, 0, 1, 2, 0), dg.Thresholds(3, 2, 1, 2, 0), dg.Thresholds(1, 2, 1, 0, 0),
               dg.Thresholds(1, 2, 1, 2, 7), dg.Thresholds(1, 1 << 16, 1, 2, 0)]:
        assert L.dualgcn_partition(ctypes.byref(c), 0, 4, 4, ctypes.byref(th), None,
                                   ctypes.byref(out)) == dg.ERR_INVALID_ARG
    # keys would not fit 63 bits
    th = dg.Thresholds(1, 60000, 1, 2, 0)
    huge = _csr(dg, nnz=(1 << 31) - 1)
    assert L.dualgcn_partition(ctypes.byref(huge), 0, 0xFFFFFFFF, 4, ctypes.byref(th), None,
                               ctypes.byref(out)) == dg.ERR_UNSUPPORTED


def test_other_entry_points_reject_null(dg):
    L = dg.lib()
    assert L.dualgcn_spmm(None, 1, 2, 4, None) == dg.ERR_INVALID_ARG
    assert L.dualgcn_spmm_act(None, 1, 2, 4, dg.RELU, None) == dg.ERR_INVALID_ARG
    assert L.dualgcn_update(None, 16, 32, 8, 32, 32, 0, None) == dg.ERR_INVALID_ARG
    assert L.dualgcn_update(16, 32, 48, 0, 32, 32, 0, None) == dg.ERR_INVALID_ARG
    assert L.dualgcn_update(16, 32, 1 << 20, 8, 48, 32, 0, None) == dg.ERR_UNSUPPORTED
    assert L.dualgcn_update(16, 32, 1 << 20, 8, 32, 32, 8, None) == dg.ERR_INVALID_ARG   # bad flag
    assert L.dualgcn_spmm_act(None, 16, 32, 8, 8, None) == dg.ERR_INVALID_ARG
    assert L.dualgcn_spmm_update(None, 16, 32, 48, None, 128, 64, dg.RELU, None) == dg.ERR_INVALID_ARG
    nbytes = ctypes.c_size_t()
    assert L.dualgcn_gcn_layer_workspace(None, 32, 32, ctypes.byref(nbytes)) == dg.ERR_INVALID_ARG
    assert L.dualgcn_gcn_layer(None, 1, 2, 3, 32, 32, 0, 256, 1 << 20, None) == dg.ERR_INVALID_ARG
    assert L.dualgcn_plan_query(None, None) == dg.ERR_INVALID_ARG
    assert L.dualgcn_plan_export(None, None, None, None) == dg.ERR_INVALID_ARG
    c = _csr(dg)
    assert L.dualgcn_arw_patterns(ctypes.byref(c), 0, 4, 4, None, None) == dg.ERR_INVALID_ARG
    huge = _csr(dg, n=1 << 30)
    assert L.dualgcn_arw_patterns(ctypes.byref(huge), 0, 1 << 10, 255, 1, None) == dg.ERR_UNSUPPORTED
    L.dualgcn_plan_destroy(None)                     # no-op


def test_plan_io_checks_arguments(dg):
    L = dg.lib()
    nbytes = ctypes.c_size_t(0)
    out = ctypes.c_void_p(5)
    assert L.dualgcn_plan_save(None, None, ctypes.byref(nbytes)) == dg.ERR_INVALID_ARG
    c = _csr(dg, n=4, nnz=4)
    assert L.dualgcn_plan_load(ctypes.byref(c), None, 0, None, ctypes.byref(out)) == dg.ERR_INVALID_ARG
    assert out.value is None
    junk = ctypes.create_string_buffer(b"NOTAPLAN" + bytes(72 + 16))
    assert L.dualgcn_plan_load(ctypes.byref(c), junk, 96, None, ctypes.byref(out)) == dg.ERR_INVALID_ARG
    # a well-formed header for another size of matrix: refused before any device use
    import struct
    hdr = b"DGCNPLAN" + struct.pack("<IIii q Q II IIIIi i Q", 1, 80, 5, 0, 4, 0, 8, 4, 1, 2, 1, 2, 0, 0, 0)
    assert len(hdr) == 80
    blob = ctypes.create_string_buffer(hdr + bytes(20), 100)
    assert L.dualgcn_plan_load(ctypes.byref(c), blob, 100, None, ctypes.byref(out)) == dg.ERR_INVALID_ARG


def test_aggregator_values_checks_arguments(dg):
    L = dg.lib()
    c = _csr(dg, rowptr=1 << 20, col=1 << 24, val=1 << 28)
    assert L.dualgcn_aggregator_values(None, 0, 0.0, 1 << 30, None) == dg.ERR_INVALID_ARG
    assert L.dualgcn_aggregator_values(ctypes.byref(c), 0, 0.0, None, None) == dg.ERR_INVALID_ARG
    assert L.dualgcn_aggregator_values(ctypes.byref(c), 3, 0.0, 1 << 30, None) == dg.ERR_INVALID_ARG
    assert L.dualgcn_aggregator_values(ctypes.byref(c), -1, 0.0, 1 << 30, None) == dg.ERR_INVALID_ARG
    assert L.dualgcn_aggregator_values(ctypes.byref(c), 0, 0.0, 1 << 24, None) == dg.ERR_INVALID_ARG


def test_training_entry_points_check_arguments(dg):
    L = dg.lib()
    # softmax cross-entropy: null pointers, empty shapes, overlapping outputs
    assert L.dualgcn_softmax_xent(None, 64, 10, 4, 1.0, 1 << 20, 1 << 24, None) == dg.ERR_INVALID_ARG
    assert L.dualgcn_softmax_xent(1 << 20, 64, 0, 4, 1.0, 1 << 24, 1 << 28, None) == dg.ERR_INVALID_ARG
    assert L.dualgcn_softmax_xent(1 << 20, 64, 10, 1 << 20, 1.0, 1 << 34, 1 << 40, None) == dg.ERR_UNSUPPORTED
    assert L.dualgcn_softmax_xent(1 << 20, 64, 10, 4, 1.0, (1 << 20) + 16, 1 << 28, None) == dg.ERR_INVALID_ARG
    # weight gradient: workspace query, shapes, flags, alignment, workspace size
    nbytes = ctypes.c_size_t()
    assert L.dualgcn_weight_grad_workspace(0, 32, 32, ctypes.byref(nbytes)) == dg.ERR_INVALID_ARG
    assert L.dualgcn_weight_grad_workspace(100, 32, 32, None) == dg.ERR_INVALID_ARG
    assert L.dualgcn_weight_grad_workspace(100, 32, 64, ctypes.byref(nbytes)) == dg.OK
    assert nbytes.value == 2 * 32 * 64 * 4                  # two 64-row chunks: two partials
    assert L.dualgcn_weight_grad_workspace(1 << 22, 256, 128, ctypes.byref(nbytes)) == dg.OK
    assert nbytes.value == 1024 * 256 * 128 * 4             # at most 1024 partials
    X, G, dW, ws = 1 << 30, 1 << 31, 1 << 32, 1 << 33
    big = 1 << 28
    assert L.dualgcn_weight_grad(None, G, dW, 100, 32, 32, 0, 0.0, None, ws, big, None) == dg.ERR_INVALID_ARG
    assert L.dualgcn_weight_grad(X, G, dW, 100, 48, 32, 0, 0.0, None, ws, big, None) == dg.ERR_UNSUPPORTED
    assert L.dualgcn_weight_grad(X, G, dW, 100, 32, 32, 1, 0.0, None, ws, big, None) == dg.ERR_INVALID_ARG
    assert L.dualgcn_weight_grad(X, G + 8, dW, 100, 32, 32, 0, 0.0, None, ws, big, None) == dg.ERR_INVALID_ARG
    assert L.dualgcn_weight_grad(X, G, dW, 100, 32, 32, 0, 0.0, None, ws + 16, big, None) == dg.ERR_INVALID_ARG
    assert L.dualgcn_weight_grad(X, G, dW, 100, 32, 32, 0, 0.0, None, ws, 16, None) == dg.ERR_INVALID_ARG
    assert L.dualgcn_weight_grad(X, G, X, 100, 32, 32, 0, 0.0, None, ws, big, None) == dg.ERR_INVALID_ARG
    assert L.dualgcn_weight_grad(X, G, dW, 100, 32, 32, 0, 0.1, dW, ws, big, None) == dg.ERR_INVALID_ARG
    # weight gradient without allocation: the same checks, no workspace
    assert L.dualgcn_weight_grad_noalloc(None, G, dW, 100, 32, 32, 0, 0.0, None, None) == dg.ERR_INVALID_ARG
    assert L.dualgcn_weight_grad_noalloc(X, G, None, 100, 32, 32, 0, 0.0, None, None) == dg.ERR_INVALID_ARG
    assert L.dualgcn_weight_grad_noalloc(X, G, dW, 0, 32, 32, 0, 0.0, None, None) == dg.ERR_INVALID_ARG
    assert L.dualgcn_weight_grad_noalloc(X, G, dW, 100, 48, 32, 0, 0.0, None, None) == dg.ERR_UNSUPPORTED
    assert L.dualgcn_weight_grad_noalloc(X, G, dW, 100, 32, 32, 1, 0.0, None, None) == dg.ERR_INVALID_ARG
    assert L.dualgcn_weight_grad_noalloc(X, G + 8, dW, 100, 32, 32, 0, 0.0, None, None) == dg.ERR_INVALID_ARG
    assert L.dualgcn_weight_grad_noalloc(X, G, X, 100, 32, 32, 0, 0.0, None, None) == dg.ERR_INVALID_ARG
    assert L.dualgcn_weight_grad_noalloc(X, G, dW, 100, 32, 32, 0, 0.1, dW, None) == dg.ERR_INVALID_ARG
    # backward data
    M, dX = 1 << 34, 1 << 35
    assert L.dualgcn_backward_data(None, 16, M, dX, 10, 32, 32, 0, None) == dg.ERR_INVALID_ARG
    assert L.dualgcn_backward_data(G, 16, M, dX, 10, 32, 48, 0, None) == dg.ERR_UNSUPPORTED
    assert L.dualgcn_backward_data(G, 16, M, dX, 10, 32, 32, 1, None) == dg.ERR_INVALID_ARG
    assert L.dualgcn_backward_data(G, 16, M, G, 10, 32, 32, 0, None) == dg.ERR_INVALID_ARG
    assert L.dualgcn_backward_data(G, 16, M, M, 10, 32, 32, 0, None) == dg.ERR_INVALID_ARG


@pytest.mark.skipif(gpu_available(), reason="checks the no-device path")
def test_valid_arguments_without_device_report_no_device(dg):
    L = dg.lib()
    c = _csr(dg)
    out = ctypes.c_void_p()
    assert L.dualgcn_partition(ctypes.byref(c), 0, 4, 4, None, None, ctypes.byref(out)) == dg.ERR_NO_DEVICE
    assert out.value is None
    assert L.dualgcn_arw_patterns(ctypes.byref(c), 0, 4, 4, 1, None) == dg.ERR_NO_DEVICE
    assert L.dualgcn_aggregator_values(ctypes.byref(c), 0, 0.0, 1 << 30, None) == dg.ERR_NO_DEVICE
    assert L.dualgcn_weight_grad_noalloc(1 << 30, 1 << 31, 1 << 32, 100, 32, 32, 0, 0.0, None,
                                          None) == dg.ERR_NO_DEVICE


def test_binding_rejects_host_tensors(dg):
    import torch
    r = torch.zeros(5, dtype=torch.int32)
    with pytest.raises(TypeError):
        dg.Plan(r, torch.zeros(0, dtype=torch.int32), torch.zeros(0))


def test_plain_c_client(dg, tmp_path):
    """The header compiles as strict C99 and a C program linked with the library runs."""
    import os
    import shutil
    import subprocess
    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        pytest.skip("no C compiler")
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    libdir = os.path.join(root, "paper_2609_01983_amd")
    exe = str(tmp_path / "abi_client")
    subprocess.run([cc, "-std=c99", "-Wall", "-Wextra", "-pedantic", "-Werror",
                    "-I", os.path.join(root, "include"),
                    os.path.join(root, "tests", "c_client", "abi_client.c"),
                    "-L", libdir, "-ldualgcn", "-Wl,-rpath," + libdir, "-o", exe],
                   check=True, capture_output=True, text=True)
    r = subprocess.run([exe], capture_output=True, text=True, timeout=60)
    assert r.returncode == 0, f"check {r.returncode} failed: {r.stdout} {r.stderr}"
    assert "c client: ok" in r.stdout
