"""The C-ABI library without a GPU: symbols, the host codebook builder, and
argument checks that must fail before any HIP call (nothing is enqueued).

Every call below carries at least one invalid argument (or n == 0), so none of
them reaches the HIP runtime; fake pointers are never dereferenced.
"""
import ctypes
import os
import re

import numpy as np
import pytest

import oracle
from paper_2110_02861_amd import bq

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
A16 = 0x10000          # a 16-byte aligned fake address, never dereferenced
MIS = 0x10004          # 4-byte aligned, not 16-byte aligned


@pytest.fixture(scope="module")
def L():
    return bq.lib()


def header_functions():
    text = open(os.path.join(ROOT, "include", "bq.h")).read()
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\s*\*?\s*(bq_\w+)\s*\(", text, re.M)))


def test_header_declares_exactly_the_exports():
    assert header_functions() == sorted(bq.EXPORTS)


def test_library_exports_every_declared_symbol(L):
    for name in header_functions():
        assert hasattr(L, name), name
    # and no C++ mangled bq entry points leak as the public API
    out = os.popen(f"nm -D --defined-only {bq.LIB_PATH}").read()
    for name in header_functions():
        assert re.search(rf"\bT {name}\b", out), name


@pytest.mark.parametrize("kind", [bq.BQ_SIGNED, bq.BQ_UNSIGNED])
def test_codebook_equals_oracle_bit_for_bit(kind):
    got = bq.bq_make_dynamic_codebook(kind)
    want = oracle.dynamic_codebook(kind)
    np.testing.assert_array_equal(got.view(np.uint32), want.view(np.uint32))


def test_codebook_errors(L):
    out = np.empty(256, np.float32)
    assert L.bq_make_dynamic_codebook(2, out.ctypes.data) == bq.BQ_ERR_ENUM
    assert L.bq_make_dynamic_codebook(0, None) == bq.BQ_ERR_NULL


def test_status_strings(L):
    for s in range(9):
        assert len(bq.status_string(s)) > 0
    assert bq.status_string(999) == "unknown status"


def test_quantize_argument_checks(L):
    q = L.bq_quantize_blockwise
    assert q(A16, A16, -1, 2048, A16, A16, None) == bq.BQ_ERR_SIZE
    for b in (0, 100, 128, 3000, 8192, -2048):
        assert q(A16, A16, 10, b, A16, A16, None) == bq.BQ_ERR_BLOCKSIZE
    assert q(None, A16, 10, 2048, A16, A16, None) == bq.BQ_ERR_NULL
    assert q(A16, None, 10, 2048, A16, A16, None) == bq.BQ_ERR_NULL
    assert q(A16, A16, 10, 2048, None, A16, None) == bq.BQ_ERR_NULL
    assert q(A16, A16, 10, 2048, A16, None, None) == bq.BQ_ERR_NULL
    assert q(A16, MIS, 10, 2048, A16, A16, None) == bq.BQ_ERR_ALIGN
    assert q(A16, A16, 10, 2048, MIS, A16, None) == bq.BQ_ERR_ALIGN
    assert q(A16, A16, 10, 2048, A16, A16 + 2, None) == bq.BQ_ERR_ALIGN
    assert q(A16 + 1, A16, 10, 2048, A16, A16, None) == bq.BQ_ERR_ALIGN
    # n == 0 is a no-op, even with NULL buffers
    assert q(None, None, 0, 2048, None, None, None) == bq.BQ_OK


def test_dequantize_argument_checks(L):
    d = L.bq_dequantize_blockwise
    assert d(A16, A16, A16, -5, 2048, A16, None) == bq.BQ_ERR_SIZE
    assert d(A16, A16, A16, 5, 1000, A16, None) == bq.BQ_ERR_BLOCKSIZE
    assert d(A16, None, A16, 5, 2048, A16, None) == bq.BQ_ERR_NULL
    assert d(A16, A16, A16, 5, 2048, None, None) == bq.BQ_ERR_NULL
    assert d(A16, MIS, A16, 5, 2048, A16, None) == bq.BQ_ERR_ALIGN
    assert d(A16, A16, A16, 5, 2048, MIS, None) == bq.BQ_ERR_ALIGN
    assert d(None, None, None, 0, 256, None, None) == bq.BQ_OK


def _tensors(*rows):
    arr = (bq.bq_tensor * len(rows))()
    for i, r in enumerate(rows):
        for k, v in r.items():
            setattr(arr[i], k, v)
    return arr


def _good_row(n=100, two=True):
    return dict(param=A16, grad=A16, state1=A16, state2=A16 if two else None, absmax1=A16,
                absmax2=A16 if two else None, numel=n)


@pytest.mark.parametrize("name", ["bq_optimizer8bit_step", "bq_optimizer8bit_step_static"])
def test_step_argument_checks(L, name):
    s = getattr(L, name)
    hp = bq.bq_hparams(1e-3, 0.9, 0.995, 1e-8, 0.0, 1)
    hp0 = bq.bq_hparams(1e-3, 0.9, 0.995, 1e-8, 0.0, 0)
    good = _tensors(_good_row())
    H = ctypes.byref(hp)
    assert s(4, 2048, 0, good, 1, H, A16, A16, None) == bq.BQ_ERR_ENUM
    assert s(-1, 2048, 0, good, 1, H, A16, A16, None) == bq.BQ_ERR_ENUM
    assert s(0, 2048, 3, good, 1, H, A16, A16, None) == bq.BQ_ERR_DTYPE
    assert s(0, 1536, 0, good, 1, H, A16, A16, None) == bq.BQ_ERR_BLOCKSIZE
    assert s(0, 2048, 0, good, -1, H, A16, A16, None) == bq.BQ_ERR_SIZE
    assert s(0, 2048, 0, None, 1, H, A16, A16, None) == bq.BQ_ERR_NULL
    assert s(0, 2048, 0, good, 1, None, A16, A16, None) == bq.BQ_ERR_NULL
    assert s(0, 2048, 0, good, 1, H, None, A16, None) == bq.BQ_ERR_NULL
    assert s(0, 2048, 0, good, 1, H, A16, None, None) == bq.BQ_ERR_NULL    # Adam needs qmap2
    assert s(1, 2048, 0, good, 1, ctypes.byref(hp0), A16, A16, None) == bq.BQ_ERR_ARG
    assert s(0, 2048, 0, good, 1, H, A16 + 2, A16, None) == bq.BQ_ERR_ALIGN
    for field in ("param", "grad", "state1", "state2", "absmax1", "absmax2"):
        row = _good_row()
        row[field] = None
        assert s(0, 2048, 1, _tensors(row), 1, H, A16, A16, None) == bq.BQ_ERR_NULL, field
    for field, val in (("param", MIS), ("grad", MIS), ("state1", MIS), ("state2", MIS),
                       ("absmax1", A16 + 2), ("absmax2", A16 + 1)):
        row = _good_row()
        row[field] = val
        assert s(0, 2048, 1, _tensors(row), 1, H, A16, A16, None) == bq.BQ_ERR_ALIGN, field
    row = _good_row()
    row["numel"] = -3
    assert s(0, 2048, 1, _tensors(row), 1, H, A16, A16, None) == bq.BQ_ERR_SIZE
    # a bad tensor later in the list is still caught before anything is enqueued
    assert s(2, 2048, 0, _tensors(_good_row(two=False), dict(_good_row(two=False), grad=None)),
             2, H, A16, None, None) == bq.BQ_ERR_NULL
    # empty work is a no-op: no tensors, or only empty tensors (NULL pointers allowed)
    assert s(0, 2048, 0, None, 0, None, None, None, None) == bq.BQ_OK
    empty = _tensors(dict(numel=0))
    assert s(0, 2048, 0, empty, 1, H, A16, A16, None) == bq.BQ_OK


def test_static_step_limits(L):
    """More non-empty tensors than the static array holds, or more tiles than
    one launch covers, are refused before any HIP call."""
    s = L.bq_optimizer8bit_step_static
    H = ctypes.byref(bq.bq_hparams(1e-3, 0.9, 0.995, 1e-8, 0.0, 1))
    many = _tensors(*[_good_row(10) for _ in range(4097)])
    assert s(0, 2048, 1, many, 4097, H, A16, A16, None) == bq.BQ_ERR_SIZE
    huge = _tensors(*[_good_row(1 << 34) for _ in range(3)])  # 3 * 2^22 tiles > 8,388,607
    assert s(0, 2048, 1, huge, 3, H, A16, A16, None) == bq.BQ_ERR_SIZE


def test_momentum_does_not_need_second_state(L):
    s = L.bq_optimizer8bit_step
    hp = bq.bq_hparams(0.1, 0.9, 0.0, 0.0, 1e-4, 1)
    # second state and map absent is fine for Momentum; misaligned grad proves
    # the call stops at validation and never launches
    row = dict(_good_row(two=False), grad=MIS)
    assert s(2, 2048, 0, _tensors(row), 1, ctypes.byref(hp), A16, None, None) == bq.BQ_ERR_ALIGN


def test_prepared_codebook_argument_checks(L):
    assert L.bq_prepare_codebook(None, A16, None) == bq.BQ_ERR_NULL
    assert L.bq_prepare_codebook(A16, None, None) == bq.BQ_ERR_NULL
    assert L.bq_prepare_codebook(A16 + 2, A16, None) == bq.BQ_ERR_ALIGN
    assert L.bq_prepare_codebook(A16, A16 + 4, None) == bq.BQ_ERR_ALIGN
    q = L.bq_quantize_blockwise_prepared
    assert q(A16, A16, -1, 2048, A16, A16, None) == bq.BQ_ERR_SIZE
    assert q(A16, A16, 10, 3000, A16, A16, None) == bq.BQ_ERR_BLOCKSIZE
    assert q(None, A16, 10, 2048, A16, A16, None) == bq.BQ_ERR_NULL
    assert q(A16 + 8, A16, 10, 2048, A16, A16, None) == bq.BQ_ERR_ALIGN
    assert q(A16, MIS, 10, 2048, A16, A16, None) == bq.BQ_ERR_ALIGN
    assert q(A16, A16, 10, 2048, A16, A16 + 1, None) == bq.BQ_ERR_ALIGN
    # more tiles than one grid of 512-thread workgroups can hold
    assert q(A16, A16, (1 << 32) * 2048, 2048, A16, A16, None) == bq.BQ_ERR_SIZE
    assert q(None, None, 0, 2048, None, None, None) == bq.BQ_OK


def test_step_plan_argument_checks(L):
    c = L.bq_step_plan_create
    h = ctypes.c_void_p(123)
    good = _tensors(_good_row())
    assert c(0, 2048, 1, good, 1, None) == bq.BQ_ERR_NULL
    assert c(6, 2048, 1, good, 1, ctypes.byref(h)) == bq.BQ_ERR_ENUM
    assert h.value is None  # the handle is cleared on every error
    assert c(0, 2048, 9, good, 1, ctypes.byref(h)) == bq.BQ_ERR_DTYPE
    assert c(0, 100, 1, good, 1, ctypes.byref(h)) == bq.BQ_ERR_BLOCKSIZE
    assert c(0, 2048, 1, good, -1, ctypes.byref(h)) == bq.BQ_ERR_SIZE
    assert c(0, 2048, 1, None, 1, ctypes.byref(h)) == bq.BQ_ERR_NULL
    assert c(0, 2048, 1, _tensors(dict(_good_row(), state2=None)), 1,
             ctypes.byref(h)) == bq.BQ_ERR_NULL
    assert c(0, 2048, 1, _tensors(dict(_good_row(), param=MIS)), 1,
             ctypes.byref(h)) == bq.BQ_ERR_ALIGN
    # tile count beyond one grid
    big = _tensors(*[dict(_good_row(), numel=(1 << 31)) for _ in range(17)])
    assert c(0, 2048, 1, big, 17, ctypes.byref(h)) == bq.BQ_ERR_SIZE
    hp = bq.bq_hparams(1e-3, 0.9, 0.995, 1e-8, 0.0, 1)
    r = L.bq_step_plan_run
    assert r(None, ctypes.byref(hp), A16, A16, None) == bq.BQ_ERR_NULL
    assert L.bq_step_plan_run_prepared(None, ctypes.byref(hp), A16, None) == bq.BQ_ERR_NULL
    assert L.bq_step_plan_run_device(None, A16, 1, A16, None) == bq.BQ_ERR_NULL
    assert L.bq_step_plan_destroy(None) == bq.BQ_OK


def test_product_path_has_no_fallback(monkeypatch, tmp_path):
    """Without the built library the binding raises instead of computing."""
    monkeypatch.setattr(bq, "LIB_PATH", str(tmp_path / "missing.so"))
    monkeypatch.setattr(bq, "_lib", None)
    with pytest.raises(RuntimeError):
        bq.lib()


def _tensors32(*rows):
    arr = (bq.bq_tensor32 * len(rows))()
    for i, r in enumerate(rows):
        for k, v in r.items():
            setattr(arr[i], k, v)
    return arr


def test_step32_argument_checks(L):
    s = L.bq_optimizer32bit_step
    hp = bq.bq_hparams(1e-3, 0.9, 0.995, 1e-8, 0.0, 1)
    hp0 = bq.bq_hparams(1e-3, 0.9, 0.995, 1e-8, 0.0, 0)
    H = ctypes.byref(hp)
    row = dict(param=A16, grad=A16, state1=A16, state2=A16, numel=100)
    good = _tensors32(row)
    assert s(4, 0, good, 1, H, None) == bq.BQ_ERR_ENUM
    assert s(0, 5, good, 1, H, None) == bq.BQ_ERR_DTYPE
    assert s(0, 0, good, -1, H, None) == bq.BQ_ERR_SIZE
    assert s(0, 0, None, 1, H, None) == bq.BQ_ERR_NULL
    assert s(0, 0, good, 1, None, None) == bq.BQ_ERR_NULL
    assert s(0, 0, good, 1, ctypes.byref(hp0), None) == bq.BQ_ERR_ARG
    assert s(0, 0, _tensors32(dict(row, state2=None)), 1, H, None) == bq.BQ_ERR_NULL
    assert s(0, 0, _tensors32(dict(row, grad=MIS)), 1, H, None) == bq.BQ_ERR_ALIGN
    assert s(0, 0, _tensors32(dict(row, state1=A16 + 8)), 1, H, None) == bq.BQ_ERR_ALIGN
    assert s(0, 0, _tensors32(dict(row, numel=-1)), 1, H, None) == bq.BQ_ERR_SIZE
    # Momentum needs no second state; empty tensors and empty lists are no-ops
    assert s(2, 0, _tensors32(dict(row, state2=None, numel=0)), 1, H, None) == bq.BQ_OK
    assert s(0, 0, None, 0, H, None) == bq.BQ_OK


def test_codebook_call_checks(L):
    out = (ctypes.c_float * 256)()
    assert L.bq_make_codebook(0, None) == bq.BQ_ERR_NULL
    assert L.bq_make_codebook(6, out) == bq.BQ_ERR_ENUM
    assert L.bq_make_codebook(-1, out) == bq.BQ_ERR_ENUM
    # the dynamic-only call keeps refusing the other kinds
    assert L.bq_make_dynamic_codebook(2, out) == bq.BQ_ERR_ENUM
    x = (ctypes.c_float * 4)(1.0, 2.0, 3.0, float("nan"))
    assert L.bq_make_quantile_codebook(None, 4, out) == bq.BQ_ERR_NULL
    assert L.bq_make_quantile_codebook(x, 4, None) == bq.BQ_ERR_NULL
    assert L.bq_make_quantile_codebook(x, 0, out) == bq.BQ_ERR_SIZE
    assert L.bq_make_quantile_codebook(x, 4, out) == bq.BQ_ERR_ARG      # NaN
    z = (ctypes.c_float * 3)(0.0, 0.0, 0.0)
    assert L.bq_make_quantile_codebook(z, 3, out) == bq.BQ_ERR_ARG      # all-zero map
    assert L.bq_make_quantile_codebook(x, 3, out) == bq.BQ_OK


def test_quantile_estimator_checks(L):
    e = L.bq_estimate_quantile_codebook
    assert e(A16, 0, A16, A16, None) == bq.BQ_ERR_SIZE
    assert e(None, 10, A16, A16, None) == bq.BQ_ERR_NULL
    assert e(A16, 10, None, A16, None) == bq.BQ_ERR_NULL
    assert e(A16, 10, A16, None, None) == bq.BQ_ERR_NULL
    assert e(A16 + 2, 10, A16, A16, None) == bq.BQ_ERR_ALIGN
    assert e(A16, 10, A16 + 4, A16, None) == bq.BQ_ERR_ALIGN
    assert e(A16, 1 << 62, A16, A16, None) == bq.BQ_ERR_SIZE
    w = L.bq_quantile_workspace_bytes
    assert w(0) == 0
    assert w(1) == 1032 + 257 * 8          # one chunk: 257 floats padded to 8 B, one group
    assert w(4096 * 64) == 64 * 257 * 4 + 257 * 8
    assert w(4096 * 64 + 1) == (65 * 257 * 4 + 7) // 8 * 8 + 2 * 257 * 8
