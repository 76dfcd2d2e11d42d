"""Property test of the C ABI's argument checks, without a GPU.

Every generated call carries at least one violation of the contract in
include/bq.h (or is an empty no-op), so it must return before any HIP call:
one of the error codes its violations map to (BQ_OK for an empty call).  Fake
pointers are never dereferenced: a call that would reach the GPU is never
generated.
"""
import ctypes

import pytest
import torch
from hypothesis import HealthCheck, assume, given, settings
from hypothesis import strategies as st

from paper_2110_02861_amd import bq

# The calls carry fake device pointers: run them only where no GPU can be
# reached, so that a gap in the model below fails as an error code here
# instead of launching.
pytestmark = pytest.mark.skipif(torch.cuda.is_available(),
                                reason="fake device pointers; runs where no GPU is visible")

A16 = 0x10000  # aligned fake address
MIS16 = 0x10004  # 4-byte aligned, not 16-byte aligned
MIS4 = 0x10002  # not 4-byte aligned
MAX_TILES = (1 << 32) // 512 - 1

SETTINGS = settings(max_examples=400, derandomize=True, deadline=None,
                    suppress_health_check=[HealthCheck.too_slow])
ptr16 = st.sampled_from(["ok", "null", "mis"])  # element arrays: 16-byte alignment
ptr4 = st.sampled_from(["ok", "null", "mis"])   # absmax and maps: 4-byte alignment
blocksizes = st.sampled_from([256, 512, 1024, 2048, 4096, 0, -2048, 100, 3000, 8192, 1 << 30])
sizes = st.one_of(st.integers(-5, 5), st.integers(-(1 << 40), 1 << 45),
                  st.sampled_from([2048, 4097, MAX_TILES * 4096 + 1]))


def addr(kind, need):
    return {"ok": A16, "null": None, "mis": MIS16 if need == 16 else MIS4}[kind]


def pointer_errors(pairs):
    """Errors of (kind, alignment) pointer arguments: NULL, then misalignment."""
    errs = set()
    for kind, _ in pairs:
        if kind == "null":
            errs.add(bq.BQ_ERR_NULL)
        elif kind == "mis":
            errs.add(bq.BQ_ERR_ALIGN)
    return errs


def valid_blocksize(b):
    return 256 <= b <= 4096 and b & (b - 1) == 0


@SETTINGS
@given(n=sizes, b=blocksizes, q=ptr4, x=ptr16, c=ptr16, a=ptr4)
def test_quantize_checks(n, b, q, x, c, a):
    errs = pointer_errors([(q, 4), (x, 16), (c, 16), (a, 4)])
    if n < 0:
        errs.add(bq.BQ_ERR_SIZE)
    if not valid_blocksize(b):
        errs.add(bq.BQ_ERR_BLOCKSIZE)
    allowed = errs | ({bq.BQ_OK} if n == 0 else set())
    assume(allowed)  # else the call is valid and would launch
    r = bq.lib().bq_quantize_blockwise(addr(q, 4), addr(x, 16), n, b, addr(c, 16), addr(a, 4),
                                       None)
    assert r in allowed, (r, allowed)


@SETTINGS
@given(n=sizes, b=blocksizes, q=ptr4, c=ptr16, a=ptr4, o=ptr16)
def test_dequantize_checks(n, b, q, c, a, o):
    errs = pointer_errors([(q, 4), (c, 16), (a, 4), (o, 16)])
    if n < 0 or (n + 4095) // 4096 > MAX_TILES:
        errs.add(bq.BQ_ERR_SIZE)
    if not valid_blocksize(b):
        errs.add(bq.BQ_ERR_BLOCKSIZE)
    allowed = errs | ({bq.BQ_OK} if n == 0 else set())
    assume(allowed)
    r = bq.lib().bq_dequantize_blockwise(addr(q, 4), addr(c, 16), addr(a, 4), n, b,
                                         addr(o, 16), None)
    assert r in allowed, (r, allowed)


row = st.fixed_dictionaries({
    "numel": st.one_of(st.integers(-3, 3), st.sampled_from([100, 4096, 1 << 44])),
    "param": ptr16, "grad": ptr16, "state1": ptr16, "state2": ptr16,
    "absmax1": ptr4, "absmax2": ptr4})


@SETTINGS
@given(opt=st.integers(-1, 7), dtype=st.integers(-1, 4), b=blocksizes,
       rows=st.lists(row, min_size=0, max_size=3), ntensors_delta=st.sampled_from([0, 0, -1]),
       tensors_null=st.booleans(), hp_kind=st.sampled_from(["ok", "null", "step0"]),
       q1=ptr4, q2=ptr4)
def test_step_checks(opt, dtype, b, rows, ntensors_delta, tensors_null, hp_kind, q1, q2):
    ntensors = len(rows) if ntensors_delta == 0 else -1
    errs = set()
    if opt not in (bq.BQ_ADAM, bq.BQ_ADAMW, bq.BQ_MOMENTUM, bq.BQ_ADAGRAD):
        errs.add(bq.BQ_ERR_ENUM)
    if dtype not in (bq.BQ_F32, bq.BQ_F16, bq.BQ_BF16):
        errs.add(bq.BQ_ERR_DTYPE)
    if not valid_blocksize(b):
        errs.add(bq.BQ_ERR_BLOCKSIZE)
    if ntensors < 0:
        errs.add(bq.BQ_ERR_SIZE)
    two = opt in (bq.BQ_ADAM, bq.BQ_ADAMW)
    if ntensors > 0:
        if tensors_null or hp_kind == "null":
            errs.add(bq.BQ_ERR_NULL)
        if hp_kind == "step0":
            errs.add(bq.BQ_ERR_ARG)
        errs |= pointer_errors([(q1, 4)] + ([(q2, 4)] if two else []))
        if not tensors_null:
            tile = 4096 if valid_blocksize(b) else 1
            for r in rows:
                if r["numel"] < 0 or r["numel"] // tile >= (2**31 - 1) // 2:
                    errs.add(bq.BQ_ERR_SIZE)
                if r["numel"] > 0:
                    ptrs = [(r["param"], 16), (r["grad"], 16), (r["state1"], 16),
                            (r["absmax1"], 4)]
                    if two:
                        ptrs += [(r["state2"], 16), (r["absmax2"], 4)]
                    errs |= pointer_errors(ptrs)
    empty = ntensors == 0 or (ntensors > 0 and all(r["numel"] == 0 for r in rows))
    allowed = errs | ({bq.BQ_OK} if empty else set())
    assume(allowed)
    arr = None
    if rows and not tensors_null:
        arr = (bq.bq_tensor * len(rows))()
        for i, r in enumerate(rows):
            arr[i].numel = r["numel"]
            for k, need in (("param", 16), ("grad", 16), ("state1", 16), ("state2", 16),
                            ("absmax1", 4), ("absmax2", 4)):
                setattr(arr[i], k, addr(r[k], need))
    hp = None if hp_kind == "null" else bq.bq_hparams(1e-3, 0.9, 0.99, 1e-8, 0.0,
                                                      0 if hp_kind == "step0" else 1)
    r = bq.lib().bq_optimizer8bit_step(opt, b, dtype, arr, ntensors,
                                       None if hp is None else ctypes.byref(hp),
                                       addr(q1, 4), addr(q2, 4), None)
    assert r in allowed, (r, allowed)
