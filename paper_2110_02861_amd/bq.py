"""ctypes binding of libbq (include/bq.h), with the C names.

Argument marshalling only: torch tensors are passed as device pointers and the
current torch stream as the HIP stream; every step of the path runs in the HIP
kernels of libbq.so.  There is no fallback: if the library is not built, or a
call returns an error, an exception is raised.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
# BQ_SANITIZE=1 selects the host-sanitized build (build.py --sanitize), for the
# CPU tests under AddressSanitizer / UndefinedBehaviorSanitizer only
LIB_PATH = (os.path.join(_PKG, "_build", "san", "libbq.so") if os.environ.get("BQ_SANITIZE") == "1"
            else os.path.join(_PKG, "libbq.so"))

BQ_OK, BQ_ERR_NULL, BQ_ERR_SIZE, BQ_ERR_BLOCKSIZE, BQ_ERR_ENUM = 0, 1, 2, 3, 4
BQ_ERR_DTYPE, BQ_ERR_ALIGN, BQ_ERR_HIP, BQ_ERR_ARG = 5, 6, 7, 8
BQ_SIGNED, BQ_UNSIGNED = 0, 1
BQ_INVERSE_SIGNED, BQ_INVERSE_UNSIGNED = 2, 3
BQ_LINEAR_SIGNED, BQ_LINEAR_UNSIGNED = 4, 5
CODEBOOKS = {"dynamic": (BQ_SIGNED, BQ_UNSIGNED),
             "inverse_dynamic": (BQ_INVERSE_SIGNED, BQ_INVERSE_UNSIGNED),
             "linear": (BQ_LINEAR_SIGNED, BQ_LINEAR_UNSIGNED)}
BQ_ADAM, BQ_ADAMW, BQ_MOMENTUM, BQ_ADAGRAD, BQ_LAMB, BQ_LARS = 0, 1, 2, 3, 4, 5
BQ_F32, BQ_F16, BQ_BF16 = 0, 1, 2
OPTIMIZERS = {"adam": BQ_ADAM, "adamw": BQ_ADAMW, "momentum": BQ_MOMENTUM,
              "adagrad": BQ_ADAGRAD, "lamb": BQ_LAMB, "lars": BQ_LARS}

EXPORTS = ("bq_make_dynamic_codebook", "bq_make_codebook", "bq_make_quantile_codebook",
           "bq_estimate_quantile_codebook", "bq_quantile_workspace_bytes",
           "bq_quantize_blockwise", "bq_dequantize_blockwise",
           "bq_optimizer8bit_step", "bq_optimizer8bit_step_static", "bq_optimizer32bit_step",
           "bq_prepare_codebook",
           "bq_quantize_blockwise_prepared",
           "bq_step_plan_create", "bq_step_plan_run", "bq_step_plan_run_prepared",
           "bq_step_plan_run_device", "bq_step_plan_destroy", "bq_status_string")
BQ_PREPARED_CODEBOOK_BYTES = 8720
BQ_QUANTILE_CHUNK = 4096


class BQError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {status_string(status)} (status {status})")


class bq_tensor(ctypes.Structure):
    _fields_ = [("param", ctypes.c_void_p), ("grad", ctypes.c_void_p),
                ("state1", ctypes.c_void_p), ("state2", ctypes.c_void_p),
                ("absmax1", ctypes.c_void_p), ("absmax2", ctypes.c_void_p),
                ("numel", ctypes.c_int64)]


class bq_tensor32(ctypes.Structure):
    _fields_ = [("param", ctypes.c_void_p), ("grad", ctypes.c_void_p),
                ("state1", ctypes.c_void_p), ("state2", ctypes.c_void_p),
                ("numel", ctypes.c_int64)]


class bq_hparams(ctypes.Structure):
    _fields_ = [("lr", ctypes.c_float), ("beta1", ctypes.c_float), ("beta2", ctypes.c_float),
                ("eps", ctypes.c_float), ("weight_decay", ctypes.c_float),
                ("step", ctypes.c_int64), ("trust_coeff", ctypes.c_float)]


_lib = None


def lib() -> ctypes.CDLL:
    """Load libbq.so (built by ``__graft_entry__.build()``); raise if absent."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is not built; run `python -m "
                               "paper_2110_02861_amd.build` (hipcc, gfx950)")
        L = ctypes.CDLL(LIB_PATH)
        P, I32, I64, I = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_int
        L.bq_make_dynamic_codebook.argtypes = [I, P]
        L.bq_make_dynamic_codebook.restype = I
        L.bq_make_codebook.argtypes = [I, P]
        L.bq_make_codebook.restype = I
        L.bq_make_quantile_codebook.argtypes = [P, I64, P]
        L.bq_make_quantile_codebook.restype = I
        L.bq_estimate_quantile_codebook.argtypes = [P, I64, P, P, P]
        L.bq_estimate_quantile_codebook.restype = I
        L.bq_quantile_workspace_bytes.argtypes = [I64]
        L.bq_quantile_workspace_bytes.restype = I64
        L.bq_quantize_blockwise.argtypes = [P, P, I64, I32, P, P, P]
        L.bq_quantize_blockwise.restype = I
        L.bq_dequantize_blockwise.argtypes = [P, P, P, I64, I32, P, P]
        L.bq_dequantize_blockwise.restype = I
        L.bq_optimizer8bit_step.argtypes = [I, I32, I, P, I32, P, P, P, P]
        L.bq_optimizer8bit_step.restype = I
        L.bq_optimizer8bit_step_static.argtypes = [I, I32, I, P, I32, P, P, P, P]
        L.bq_optimizer8bit_step_static.restype = I
        L.bq_optimizer32bit_step.argtypes = [I, I, P, I32, P, P]
        L.bq_optimizer32bit_step.restype = I
        L.bq_prepare_codebook.argtypes = [P, P, P]
        L.bq_prepare_codebook.restype = I
        L.bq_quantize_blockwise_prepared.argtypes = [P, P, I64, I32, P, P, P]
        L.bq_quantize_blockwise_prepared.restype = I
        L.bq_step_plan_create.argtypes = [I, I32, I, P, I32, ctypes.POINTER(ctypes.c_void_p)]
        L.bq_step_plan_create.restype = I
        L.bq_step_plan_run.argtypes = [P, P, P, P, P]
        L.bq_step_plan_run.restype = I
        L.bq_step_plan_run_prepared.argtypes = [P, P, P, P]
        L.bq_step_plan_run_prepared.restype = I
        L.bq_step_plan_run_device.argtypes = [P, P, I32, P, P]
        L.bq_step_plan_run_device.restype = I
        L.bq_step_plan_destroy.argtypes = [P]
        L.bq_step_plan_destroy.restype = I
        L.bq_status_string.argtypes = [I]
        L.bq_status_string.restype = ctypes.c_char_p
        _lib = L
    return _lib


def status_string(s: int) -> str:
    return lib().bq_status_string(int(s)).decode()


def _check(status: int, where: str) -> None:
    if status != BQ_OK:
        raise BQError(status, where)


def _dev_ptr(t, name):
    import torch
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{name} must be a GPU torch tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if t.get_device() != torch.cuda.current_device():
        # the C calls run on the current device
        raise ValueError(f"{name} is on cuda:{t.get_device()}, the current device is "
                         f"cuda:{torch.cuda.current_device()}")
    return t.data_ptr()


def _map_ptr(q, name):
    """A codebook: 256 fp32 values on the current device."""
    import torch
    if not isinstance(q, torch.Tensor) or q.dtype != torch.float32 or q.numel() != 256:
        raise TypeError(f"{name} must be a tensor of 256 fp32 values")
    return _dev_ptr(q, name)


def _stream(stream):
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream


def bq_make_dynamic_codebook(kind: int) -> np.ndarray:
    """Host call: the 256-entry signed (0) or unsigned (1) dynamic codebook."""
    out = np.empty(256, np.float32)
    _check(lib().bq_make_dynamic_codebook(int(kind), out.ctypes.data), "bq_make_dynamic_codebook")
    return out


def bq_make_codebook(kind: int) -> np.ndarray:
    """Host call: any fixed codebook (BQ_SIGNED ... BQ_LINEAR_UNSIGNED)."""
    out = np.empty(256, np.float32)
    _check(lib().bq_make_codebook(int(kind), out.ctypes.data), "bq_make_codebook")
    return out


def bq_estimate_quantile_codebook(x, out=None, workspace=None, stream=None):
    """GPU quantile map of a device fp32 tensor (App. F.2, App. G); returns the
    device map (256 fp32).  The workspace (bq_quantile_workspace_bytes) is
    allocated here by torch unless given."""
    import torch
    n = x.numel()
    if x.dtype != torch.float32:
        raise TypeError("x must be fp32")
    nbytes = max(8, int(lib().bq_quantile_workspace_bytes(n)))
    if workspace is None:
        workspace = torch.empty(nbytes // 8, dtype=torch.float64, device=x.device)
    elif workspace.numel() * workspace.element_size() < nbytes:
        raise ValueError(f"workspace holds {workspace.numel() * workspace.element_size()} "
                         f"bytes, needs {nbytes}")
    if out is None:
        out = torch.empty(256, dtype=torch.float32, device=x.device)
    elif out.dtype != torch.float32 or out.numel() != 256:
        raise TypeError("out must be a tensor of 256 fp32 values")
    _check(lib().bq_estimate_quantile_codebook(_dev_ptr(x, "x") if n else None, n,
                                               _dev_ptr(workspace, "workspace"),
                                               _dev_ptr(out, "out"), _stream(stream)),
           "bq_estimate_quantile_codebook")
    return out


def bq_make_quantile_codebook(sample) -> np.ndarray:
    """Host call: the quantile map of a host fp32 sample (App. F.2)."""
    x = np.ascontiguousarray(sample, dtype=np.float32).ravel()
    out = np.empty(256, np.float32)
    _check(lib().bq_make_quantile_codebook(x.ctypes.data if x.size else None, x.size,
                                           out.ctypes.data), "bq_make_quantile_codebook")
    return out


def bq_quantize_blockwise(qmap, x, blocksize: int, codes=None, absmax=None, stream=None):
    """codes (uint8, like x) and absmax (fp32, ceil(n/B)) of the GPU tensor x."""
    import torch
    n = x.numel()
    if codes is None:
        codes = torch.empty(n, dtype=torch.uint8, device=x.device)
    if absmax is None:
        absmax = torch.empty((n + blocksize - 1) // blocksize, dtype=torch.float32,
                             device=x.device)
    if x.dtype != torch.float32 or codes.dtype != torch.uint8 or absmax.dtype != torch.float32:
        raise TypeError("x fp32, codes uint8, absmax fp32")
    if codes.numel() < n or absmax.numel() < (n + blocksize - 1) // blocksize:
        raise ValueError("output buffers too small")
    _check(lib().bq_quantize_blockwise(_map_ptr(qmap, "qmap"), _dev_ptr(x, "x"), n,
                                       int(blocksize), _dev_ptr(codes, "codes"),
                                       _dev_ptr(absmax, "absmax"), _stream(stream)),
           "bq_quantize_blockwise")
    return codes, absmax


def bq_dequantize_blockwise(qmap, codes, absmax, blocksize: int, out=None, stream=None):
    import torch
    n = codes.numel()
    if out is None:
        out = torch.empty(n, dtype=torch.float32, device=codes.device)
    if codes.dtype != torch.uint8 or absmax.dtype != torch.float32 or out.dtype != torch.float32:
        raise TypeError("codes uint8, absmax fp32, out fp32")
    if out.numel() < n or absmax.numel() < (n + blocksize - 1) // blocksize:
        raise ValueError("buffers too small")
    _check(lib().bq_dequantize_blockwise(_map_ptr(qmap, "qmap"), _dev_ptr(codes, "codes"),
                                         _dev_ptr(absmax, "absmax"), n, int(blocksize),
                                         _dev_ptr(out, "out"), _stream(stream)),
           "bq_dequantize_blockwise")
    return out


def _grad_torch_dtype(grad_dtype):
    import torch
    return {BQ_F32: torch.float32, BQ_F16: torch.float16,
            BQ_BF16: torch.bfloat16}.get(int(grad_dtype))


def check_step_tensors(opt, blocksize: int, grad_dtype: int, tensors) -> None:
    """Sizes, dtypes and device of a step's (param, grad, state1, state2,
    absmax1, absmax2) tuples.  The C ABI takes plain pointers and cannot see
    them: a state or absmax array shorter than its param would be written
    past its end.  Raises ValueError / TypeError."""
    import torch
    if isinstance(opt, str):
        opt = OPTIMIZERS[opt]
    two = int(opt) in (BQ_ADAM, BQ_ADAMW, BQ_LAMB)
    gdt = _grad_torch_dtype(grad_dtype)
    cur = torch.cuda.current_device()
    B = int(blocksize)
    for i, (p, g, s1, s2, a1, a2) in enumerate(tensors):
        n = p.numel()
        want = [(p, "param", torch.float32, n), (g, "grad", gdt, n), (s1, "state1", torch.uint8, n)]
        if B > 0:
            want.append((a1, "absmax1", torch.float32, (n + B - 1) // B))
        if two:
            want.append((s2, "state2", torch.uint8, n))
            if B > 0:
                want.append((a2, "absmax2", torch.float32, (n + B - 1) // B))
        for t, name, dtype, size in want:
            if not isinstance(t, torch.Tensor):
                raise TypeError(f"tensor {i}: {name} must be a torch tensor")
            if dtype is not None and t.dtype != dtype:
                raise TypeError(f"tensor {i}: {name} must be {dtype}, got {t.dtype}")
            if t.numel() < size:
                raise ValueError(f"tensor {i}: {name} holds {t.numel()} elements, needs {size}")
            if t.is_cuda and t.get_device() != cur:
                raise ValueError(f"tensor {i}: {name} is on cuda:{t.get_device()}, the current "
                                 f"device is cuda:{cur}")


def make_tensor_array(tensors):
    """Pack (param, grad, state1, state2, absmax1, absmax2) tuples of GPU
    tensors (state2 / absmax2 may be None) into a ctypes bq_tensor array."""
    arr = (bq_tensor * max(1, len(tensors)))()
    for i, (p, g, s1, s2, a1, a2) in enumerate(tensors):
        arr[i].param = _dev_ptr(p, "param")
        arr[i].grad = _dev_ptr(g, "grad")
        arr[i].state1 = _dev_ptr(s1, "state1")
        arr[i].state2 = None if s2 is None else _dev_ptr(s2, "state2")
        arr[i].absmax1 = _dev_ptr(a1, "absmax1")
        arr[i].absmax2 = None if a2 is None else _dev_ptr(a2, "absmax2")
        arr[i].numel = p.numel()
    return arr


def bq_optimizer8bit_step(opt, blocksize: int, grad_dtype: int, tensors, hp: dict, qmap1,
                          qmap2=None, stream=None):
    """One fused 8-bit step over a list of tensors (see make_tensor_array), or
    over a prebuilt ``(bq_tensor array, count)`` pair."""
    if isinstance(opt, str):
        opt = OPTIMIZERS[opt]
    if isinstance(tensors, tuple) and len(tensors) == 2 and isinstance(tensors[1], int):
        arr, count = tensors  # prebuilt by the caller, who vouches for the sizes
    else:
        check_step_tensors(opt, blocksize, grad_dtype, tensors)
        arr, count = make_tensor_array(tensors), len(tensors)
    h = _hparams(hp)
    _check(lib().bq_optimizer8bit_step(int(opt), int(blocksize), int(grad_dtype), arr, count,
                                       ctypes.byref(h), _map_ptr(qmap1, "qmap1"),
                                       None if qmap2 is None else _map_ptr(qmap2, "qmap2"),
                                       _stream(stream)),
           "bq_optimizer8bit_step")


def bq_optimizer8bit_step_static(opt, blocksize: int, grad_dtype: int, tensors, hp: dict,
                                 qmap1, qmap2=None, stream=None):
    """bq_optimizer8bit_step through the library's static device array (no
    allocation; calls on one GPU must not overlap)."""
    if isinstance(opt, str):
        opt = OPTIMIZERS[opt]
    if isinstance(tensors, tuple) and len(tensors) == 2 and isinstance(tensors[1], int):
        arr, count = tensors  # prebuilt by the caller, who vouches for the sizes
    else:
        check_step_tensors(opt, blocksize, grad_dtype, tensors)
        arr, count = make_tensor_array(tensors), len(tensors)
    h = _hparams(hp)
    _check(lib().bq_optimizer8bit_step_static(
        int(opt), int(blocksize), int(grad_dtype), arr, count, ctypes.byref(h),
        _map_ptr(qmap1, "qmap1"), None if qmap2 is None else _map_ptr(qmap2, "qmap2"),
        _stream(stream)), "bq_optimizer8bit_step_static")


def make_tensor32_array(tensors):
    """Pack (param, grad, state1, state2) tuples of GPU tensors (state2 may be
    None) into a ctypes bq_tensor32 array."""
    arr = (bq_tensor32 * max(1, len(tensors)))()
    for i, (p, g, m, v) in enumerate(tensors):
        arr[i].param = _dev_ptr(p, "param")
        arr[i].grad = _dev_ptr(g, "grad")
        arr[i].state1 = _dev_ptr(m, "state1")
        arr[i].state2 = None if v is None else _dev_ptr(v, "state2")
        arr[i].numel = p.numel()
    return arr


def bq_optimizer32bit_step(opt, grad_dtype: int, tensors, hp: dict, stream=None):
    """One step with fp32 states over (param, grad, state1, state2) tuples."""
    import torch
    if isinstance(opt, str):
        opt = OPTIMIZERS[opt]
    two = int(opt) in (BQ_ADAM, BQ_ADAMW)
    gdt = _grad_torch_dtype(grad_dtype)
    cur = torch.cuda.current_device()
    for i, (p, g, m, v) in enumerate(tensors):
        n = p.numel()
        want = [(p, "param", torch.float32), (g, "grad", gdt), (m, "state1", torch.float32)]
        if two:
            want.append((v, "state2", torch.float32))
        for t, name, dtype in want:
            if not isinstance(t, torch.Tensor):
                raise TypeError(f"tensor {i}: {name} must be a torch tensor")
            if dtype is not None and t.dtype != dtype:
                raise TypeError(f"tensor {i}: {name} must be {dtype}, got {t.dtype}")
            if t.numel() < n:
                raise ValueError(f"tensor {i}: {name} holds {t.numel()} elements, needs {n}")
            if t.is_cuda and t.get_device() != cur:
                raise ValueError(f"tensor {i}: {name} is on cuda:{t.get_device()}, the current "
                                 f"device is cuda:{cur}")
    arr = make_tensor32_array(tensors)
    h = _hparams(hp)
    _check(lib().bq_optimizer32bit_step(int(opt), int(grad_dtype), arr, len(tensors),
                                        ctypes.byref(h), _stream(stream)),
           "bq_optimizer32bit_step")


def _hparams(hp: dict) -> bq_hparams:
    return bq_hparams(hp["lr"], hp["beta1"], hp.get("beta2", 0.0), hp.get("eps", 0.0),
                      hp.get("wd", hp.get("weight_decay", 0.0)), int(hp["step"]),
                      hp.get("trust", 0.0))


def bq_prepare_codebook(qmap, prepared=None, stream=None):
    """Decision tables of a device codebook into a device uint8 buffer of
    BQ_PREPARED_CODEBOOK_BYTES (allocated here by torch if not given)."""
    import torch
    if prepared is None:
        prepared = torch.empty(BQ_PREPARED_CODEBOOK_BYTES, dtype=torch.uint8, device=qmap.device)
    if prepared.numel() < BQ_PREPARED_CODEBOOK_BYTES:
        raise ValueError("prepared buffer too small")
    _check(lib().bq_prepare_codebook(_map_ptr(qmap, "qmap"), _dev_ptr(prepared, "prepared"),
                                     _stream(stream)), "bq_prepare_codebook")
    return prepared


def bq_quantize_blockwise_prepared(prepared, x, blocksize: int, codes=None, absmax=None,
                                   stream=None):
    import torch
    n = x.numel()
    if codes is None:
        codes = torch.empty(n, dtype=torch.uint8, device=x.device)
    if absmax is None:
        absmax = torch.empty((n + blocksize - 1) // blocksize, dtype=torch.float32,
                             device=x.device)
    if x.dtype != torch.float32 or codes.dtype != torch.uint8 or absmax.dtype != torch.float32:
        raise TypeError("x fp32, codes uint8, absmax fp32")
    if codes.numel() < n or absmax.numel() < (n + blocksize - 1) // blocksize:
        raise ValueError("output buffers too small")
    if prepared.numel() * prepared.element_size() < BQ_PREPARED_CODEBOOK_BYTES:
        raise ValueError(f"prepared codebook: need {BQ_PREPARED_CODEBOOK_BYTES} bytes")
    _check(lib().bq_quantize_blockwise_prepared(_dev_ptr(prepared, "prepared"), _dev_ptr(x, "x"),
                                                n, int(blocksize), _dev_ptr(codes, "codes"),
                                                _dev_ptr(absmax, "absmax"), _stream(stream)),
           "bq_quantize_blockwise_prepared")
    return codes, absmax


def prepare_codebook_pair(qmap1, qmap2=None, stream=None):
    """Both codebooks of an optimizer prepared back to back in one device
    buffer (bq_prepare_codebook twice), as bq_step_plan_run_prepared reads
    them: map 1's tables, then map 2's (absent for one-state optimizers)."""
    import torch
    prepared = torch.empty(2 * BQ_PREPARED_CODEBOOK_BYTES, dtype=torch.uint8,
                           device=qmap1.device)
    bq_prepare_codebook(qmap1, prepared[:BQ_PREPARED_CODEBOOK_BYTES], stream)
    if qmap2 is not None:
        bq_prepare_codebook(qmap2, prepared[BQ_PREPARED_CODEBOOK_BYTES:], stream)
    return prepared


class StepPlan:
    """bq_step_plan_create / bq_step_plan_run / bq_step_plan_destroy.

    The plan holds device pointers to the given tensors.  By default this
    object keeps references to them, so they stay allocated while the plan
    lives.  keep=False drops those references: the caller must then check,
    before every run, that the same storages (pointers and sizes) are still
    the live tensors (the drop-in optimizers do)."""

    def __init__(self, opt, blocksize: int, grad_dtype: int, tensors, keep: bool = True):
        if isinstance(opt, str):
            opt = OPTIMIZERS[opt]
        self._keep = [t for row in tensors for t in row if t is not None] if keep else []
        check_step_tensors(opt, blocksize, grad_dtype, tensors)
        arr = make_tensor_array(tensors)
        h = ctypes.c_void_p()
        _check(lib().bq_step_plan_create(int(opt), int(blocksize), int(grad_dtype), arr,
                                         len(tensors), ctypes.byref(h)), "bq_step_plan_create")
        self._h = h
        self._two = opt in (BQ_ADAM, BQ_ADAMW, BQ_LAMB)

    def run(self, hp: dict, qmap1, qmap2=None, stream=None):
        h = _hparams(hp)
        _check(lib().bq_step_plan_run(self._h, ctypes.byref(h), _map_ptr(qmap1, "qmap1"),
                                      None if qmap2 is None else _map_ptr(qmap2, "qmap2"),
                                      _stream(stream)), "bq_step_plan_run")

    def run_prepared(self, hp: dict, prepared, stream=None):
        """One run with codebooks prepared beforehand (prepare_codebook_pair)."""
        import torch
        need = (2 if self._two else 1) * BQ_PREPARED_CODEBOOK_BYTES
        if prepared.dtype != torch.uint8 or prepared.numel() < need:
            raise ValueError(f"prepared codebooks: need {need} uint8 bytes")
        h = _hparams(hp)
        _check(lib().bq_step_plan_run_prepared(self._h, ctypes.byref(h),
                                               _dev_ptr(prepared, "prepared"), _stream(stream)),
               "bq_step_plan_run_prepared")

    def run_device(self, hp_device, prepared, advance: bool = True, stream=None):
        """One run whose hyperparameters are read from device memory when it
        executes (hp_device: device_hparams); capturable into a graph."""
        import torch
        need = (2 if self._two else 1) * BQ_PREPARED_CODEBOOK_BYTES
        if prepared.dtype != torch.uint8 or prepared.numel() < need:
            raise ValueError(f"prepared codebooks: need {need} uint8 bytes")
        if hp_device.dtype != torch.uint8 or hp_device.numel() != ctypes.sizeof(bq_hparams):
            raise ValueError("hp_device must come from device_hparams()")
        _check(lib().bq_step_plan_run_device(self._h, _dev_ptr(hp_device, "hp_device"),
                                             1 if advance else 0,
                                             _dev_ptr(prepared, "prepared"), _stream(stream)),
               "bq_step_plan_run_device")

    def is_open(self) -> bool:
        return getattr(self, "_h", None) is not None and self._h.value is not None

    def close(self):
        if getattr(self, "_h", None) is not None and self._h.value is not None:
            lib().bq_step_plan_destroy(self._h)
        self._h = None
        self._keep = []

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def bq_step_plan_create(opt, blocksize, grad_dtype, tensors):
    return StepPlan(opt, blocksize, grad_dtype, tensors)


def bq_step_plan_run(plan: StepPlan, hp: dict, qmap1, qmap2=None, stream=None):
    plan.run(hp, qmap1, qmap2, stream)


def bq_step_plan_run_prepared(plan: StepPlan, hp: dict, prepared, stream=None):
    plan.run_prepared(hp, prepared, stream)


def bq_step_plan_run_device(plan: StepPlan, hp_device, prepared, advance=True, stream=None):
    plan.run_device(hp_device, prepared, advance, stream)


def device_hparams(hp: dict, device=None):
    """A bq_hparams packed into a device uint8 tensor, for run_device.  Start
    from step 0 with advance=True for a first step."""
    import torch
    h = _hparams(dict(hp, step=hp.get("step", 0)))
    raw = ctypes.string_at(ctypes.addressof(h), ctypes.sizeof(h))
    t = torch.frombuffer(bytearray(raw), dtype=torch.uint8)
    return t.to("cuda" if device is None else device)


def read_device_hparams(t) -> dict:
    """The fields of a device bq_hparams (as written by device_hparams)."""
    h = bq_hparams.from_buffer_copy(bytes(t.cpu().numpy().tobytes()))
    return dict(lr=h.lr, beta1=h.beta1, beta2=h.beta2, eps=h.eps, wd=h.weight_decay,
                step=h.step, trust=h.trust_coeff)


def bq_step_plan_destroy(plan: StepPlan):
    plan.close()
