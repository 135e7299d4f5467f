"""ctypes binding of libf3s.so: argument marshalling only.

Every step of the operator runs in the HIP library; this module passes device
pointers, sizes and the current HIP stream.  torch is used for device memory
and streams.  A missing or unloadable library is an error: there is no
fallback path of any kind.
"""
import ctypes
import math
import os

import torch  # noqa: F401  (loads torch's HIP runtime before libf3s.so; see _load)

from . import build as _build

F3S_OK = 0
_STATUS = {0: "F3S_OK", 1: "F3S_ERR_INVALID_VALUE", 2: "F3S_ERR_INVALID_CSR",
           3: "F3S_ERR_UNSUPPORTED", 4: "F3S_ERR_OUT_OF_MEMORY", 5: "F3S_ERR_HIP",
           6: "F3S_ERR_TOO_LARGE"}


class F3SError(RuntimeError):
    def __init__(self, code, what):
        self.code = code
        super().__init__(f"{what}: {_STATUS.get(code, code)}")


class PlanInfo(ctypes.Structure):
    _fields_ = [
        ("N", ctypes.c_int32), ("n_windows", ctypes.c_int32),
        ("nnz_csr", ctypes.c_int64), ("nnz", ctypes.c_int64),
        ("n_unique", ctypes.c_int64), ("n_blocks", ctypes.c_int64),
        ("max_blocks", ctypes.c_int32), ("piece_blocks", ctypes.c_int32),
        ("n_items", ctypes.c_int32), ("n_split", ctypes.c_int32),
        ("n_pieces", ctypes.c_int32), ("flags", ctypes.c_int32),
        ("bsb_bytes", ctypes.c_int64), ("device_bytes", ctypes.c_int64),
        ("build_ms", ctypes.c_double),
    ]

    def as_dict(self):
        return {k: getattr(self, k) for k, _ in self._fields_}


_LIB = None


def _hip_runtimes_mapped():
    paths = set()
    try:
        with open("/proc/self/maps") as f:
            for line in f:
                if "libamdhip64" in line:
                    paths.add(os.path.realpath(line.split()[-1]))
    except OSError:
        pass
    return paths


def load_library():
    """Load libf3s.so (raises if it is missing or not loadable).

    torch is imported first so that its HIP runtime is the one libf3s.so
    binds to (both carry the soname libamdhip64.so.7); a second runtime in
    the process would make torch's stream handles meaningless to the library.
    """
    global _LIB
    if _LIB is not None:
        return _LIB
    if not os.path.exists(_build.LIB):
        raise RuntimeError(
            f"{_build.LIB} is missing: build it with "
            "`python -c 'import __graft_entry__ as g; g.build()'`")
    L = ctypes.CDLL(_build.LIB)
    runtimes = _hip_runtimes_mapped()
    if len(runtimes) > 1:
        raise RuntimeError(f"two HIP runtimes mapped in one process: {sorted(runtimes)}")
    vp, i32 = ctypes.c_void_p, ctypes.c_int32
    L.f3s_plan.argtypes = [vp, vp, i32]
    L.f3s_plan.restype = vp
    L.f3s_plan_workspace_bytes.argtypes = [i32, ctypes.c_int64]
    L.f3s_plan_workspace_bytes.restype = ctypes.c_size_t
    L.f3s_plan_ws.argtypes = [vp, vp, i32, vp, ctypes.c_size_t]
    L.f3s_plan_ws.restype = vp
    L.f3s_plan_segments.argtypes = [vp, vp, i32, vp, i32]
    L.f3s_plan_segments.restype = vp
    L.f3s_plan_window_rows.argtypes = [vp, vp]
    L.f3s_plan_window_rows.restype = ctypes.c_int
    L.f3s_run.argtypes = [vp, vp, vp, vp, vp, i32, ctypes.c_float, vp]
    L.f3s_run.restype = ctypes.c_int
    L.f3s_run_mh.argtypes = [vp, vp, vp, vp, vp, i32, i32, ctypes.c_float, vp]
    L.f3s_run_mh.restype = ctypes.c_int
    L.f3s_forward.argtypes = [vp, vp, vp, vp, vp, vp, i32, i32, ctypes.c_float, vp]
    L.f3s_forward.restype = ctypes.c_int
    L.f3s_forward_typed.argtypes = [vp, vp, vp, vp, i32, vp, i32, vp, i32, i32,
                                    ctypes.c_float, vp]
    L.f3s_forward_typed.restype = ctypes.c_int
    L.f3s_plan_transpose.argtypes = [vp]
    L.f3s_plan_transpose.restype = vp
    L.f3s_plan_transpose_workspace_bytes.argtypes = [vp]
    L.f3s_plan_transpose_workspace_bytes.restype = ctypes.c_size_t
    L.f3s_plan_transpose_ws.argtypes = [vp, vp, ctypes.c_size_t]
    L.f3s_plan_transpose_ws.restype = vp
    L.f3s_backward.argtypes = [vp, vp] + [vp] * 10 + [i32, i32, ctypes.c_float, vp]
    L.f3s_backward.restype = ctypes.c_int
    L.f3s_backward_typed.argtypes = ([vp, vp, vp, vp, vp, i32] + [vp] * 7 +
                                     [i32, i32, ctypes.c_float, vp])
    L.f3s_backward_typed.restype = ctypes.c_int
    L.f3s_backward_noalloc.argtypes = ([vp, vp, vp, vp, vp, i32] + [vp] * 6 +
                                       [i32, i32, ctypes.c_float, vp])
    L.f3s_backward_noalloc.restype = ctypes.c_int
    L.f3s_backward_noalloc_max_records.argtypes = []
    L.f3s_backward_noalloc_max_records.restype = ctypes.c_int64
    L.f3s_probe_read.argtypes = [vp, ctypes.c_size_t, vp, vp]
    L.f3s_probe_read.restype = ctypes.c_int
    L.f3s_probe_copy.argtypes = [vp, vp, ctypes.c_size_t, vp]
    L.f3s_probe_copy.restype = ctypes.c_int
    L.f3s_probe_write.argtypes = [vp, ctypes.c_size_t, ctypes.c_uint32, vp]
    L.f3s_probe_write.restype = ctypes.c_int
    L.f3s_probe_gather.argtypes = [vp, vp, vp, vp, vp, i32, vp]
    L.f3s_probe_gather.restype = ctypes.c_int
    L.f3s_probe_gather_lds.argtypes = [vp, vp, vp, vp, vp, i32, vp]
    L.f3s_probe_gather_lds.restype = ctypes.c_int
    L.f3s_probe_rows.argtypes = [vp, ctypes.c_int64, i32, i32, i32, i32, vp, vp]
    L.f3s_probe_rows.restype = ctypes.c_int
    L.f3s_run_trace.argtypes = [vp, vp, vp, vp, vp, i32, ctypes.c_float, vp, ctypes.c_size_t,
                                vp]
    L.f3s_run_trace.restype = ctypes.c_int
    L.f3s_wall_clock_khz.argtypes = [i32]
    L.f3s_wall_clock_khz.restype = ctypes.c_int32
    L.f3s_destroy.argtypes = [vp]
    L.f3s_destroy.restype = None
    L.f3s_plan_info.argtypes = [vp, ctypes.POINTER(PlanInfo)]
    L.f3s_plan_info.restype = ctypes.c_int
    L.f3s_plan_export.argtypes = [vp, vp, vp, vp, vp, vp]
    L.f3s_plan_export.restype = ctypes.c_int
    L.f3s_last_error.argtypes = []
    L.f3s_last_error.restype = ctypes.c_int
    L.f3s_status_string.argtypes = [ctypes.c_int]
    L.f3s_status_string.restype = ctypes.c_char_p
    _LIB = L
    return L


def status_string(code):
    return load_library().f3s_status_string(int(code)).decode()


def _check_device_tensor(t, name, dtype, device=None):
    """A contiguous device tensor of `dtype`, on `device` when one is given
    (the library writes through the raw pointer, so a tensor on another
    device or of another size is never handed to it)."""
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{name} must be a device tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    if device is not None and t.device != device:
        raise ValueError(f"{name} is on {t.device}, the operands on {device}")


def _qkv_shape(Q):
    """Shape of a one-head [N, d] or multi-head [N, H, d] operand."""
    if not isinstance(Q, torch.Tensor) or Q.dim() not in (2, 3):
        raise ValueError("Q must be [N, d] or [N, H, d]")
    return tuple(Q.shape)


class Plan:
    """f3s_plan on a device CSR (int32 row_ptr[N+1], int32 col_idx[nnz])."""

    @classmethod
    def _from_handle(cls, h, device, N):
        self = cls.__new__(cls)
        self._h = h
        self.device = device
        self.N = int(N)
        self.info = self._info()
        return self

    @classmethod
    def segments(cls, row_ptr, col_idx, N, seg_ptr):
        """f3s_plan_segments: windows aligned to the graphs of a batch, graph g
        holding rows seg_ptr[g] .. seg_ptr[g+1] - 1 (seg_ptr: host sequence of
        ints, first 0, last N)."""
        import numpy as np
        L = load_library()
        _check_device_tensor(row_ptr, "row_ptr", torch.int32)
        _check_device_tensor(col_idx, "col_idx", torch.int32)
        if row_ptr.numel() != int(N) + 1:
            raise ValueError("row_ptr must hold N + 1 entries")
        seg = np.ascontiguousarray(seg_ptr, dtype=np.int32)
        if seg.ndim != 1 or seg.size < 1:
            raise ValueError("seg_ptr must be a non-empty 1-D sequence")
        ci = col_idx.data_ptr() if col_idx.numel() else None
        with torch.cuda.device(row_ptr.device):
            torch.cuda.current_stream().synchronize()
            h = L.f3s_plan_segments(row_ptr.data_ptr(), ci, int(N),
                                    seg.ctypes.data_as(ctypes.c_void_p), int(seg.size - 1))
        if not h:
            raise F3SError(L.f3s_last_error(), "f3s_plan_segments")
        return Plan._from_handle(h, row_ptr.device, N)

    def window_rows(self):
        """First row of every window, then N (host numpy int32)."""
        import numpy as np
        wr = np.empty(self.info["n_windows"] + 1, dtype=np.int32)
        rc = load_library().f3s_plan_window_rows(self.handle,
                                                 wr.ctypes.data_as(ctypes.c_void_p))
        if rc != F3S_OK:
            raise F3SError(rc, "f3s_plan_window_rows")
        return wr

    def transpose(self):
        """Plan of the transposed pattern (f3s_plan_transpose_ws, its scratch
        lent from torch's caching allocator)."""
        L = load_library()
        with torch.cuda.device(self.device):
            torch.cuda.current_stream().synchronize()
            nbytes = L.f3s_plan_transpose_workspace_bytes(self.handle)
            ws = torch.empty(nbytes, dtype=torch.uint8, device=self.device)
            h = L.f3s_plan_transpose_ws(self.handle, ws.data_ptr(), nbytes)
            del ws
        if not h:
            raise F3SError(L.f3s_last_error(), "f3s_plan_transpose_ws")
        return Plan._from_handle(h, self.device, self.N)

    def __init__(self, row_ptr, col_idx, N):
        L = load_library()
        _check_device_tensor(row_ptr, "row_ptr", torch.int32)
        _check_device_tensor(col_idx, "col_idx", torch.int32)
        if row_ptr.numel() != int(N) + 1:
            raise ValueError("row_ptr must hold N + 1 entries")
        ci = col_idx.data_ptr() if col_idx.numel() else None
        with torch.cuda.device(row_ptr.device):
            torch.cuda.current_stream().synchronize()
            # the build's scratch from torch's caching allocator (the build is
            # synchronous: the memory is free again when the call returns)
            nbytes = L.f3s_plan_workspace_bytes(int(N), col_idx.numel())
            if nbytes:
                ws = torch.empty(nbytes, dtype=torch.uint8, device=row_ptr.device)
                h = L.f3s_plan_ws(row_ptr.data_ptr(), ci, int(N), ws.data_ptr(), nbytes)
                del ws
            else:
                h = L.f3s_plan(row_ptr.data_ptr(), ci, int(N))
        if not h:
            raise F3SError(L.f3s_last_error(), "f3s_plan")
        self._h = h
        self.device = row_ptr.device
        self.N = int(N)
        self.info = self._info()

    def _info(self):
        inf = PlanInfo()
        rc = load_library().f3s_plan_info(self._h, ctypes.byref(inf))
        if rc != F3S_OK:
            raise F3SError(rc, "f3s_plan_info")
        return inf.as_dict()

    @property
    def handle(self):
        if self._h is None:
            raise RuntimeError("plan was destroyed")
        return self._h

    def export(self):
        """The plan's arrays copied to host numpy arrays."""
        import numpy as np
        inf = self.info
        T, B = inf["n_windows"], inf["n_blocks"]
        blk_off = np.empty(T + 1, dtype=np.int32)
        cols = np.empty(max(16 * B, 1), dtype=np.int32)
        mask = np.empty(max(8 * B, 1), dtype=np.uint32)
        items = np.empty(max(4 * inf["n_items"], 1), dtype=np.int32)
        merges = np.empty(max(3 * inf["n_split"], 1), dtype=np.int32)
        ptr = lambda a: a.ctypes.data_as(ctypes.c_void_p)
        rc = load_library().f3s_plan_export(self.handle, ptr(blk_off), ptr(cols), ptr(mask),
                                            ptr(items), ptr(merges))
        if rc != F3S_OK:
            raise F3SError(rc, "f3s_plan_export")
        return dict(blk_off=blk_off, cols=cols[: 16 * B], mask=mask[: 8 * B],
                    items=items[: 4 * inf["n_items"]].reshape(-1, 4),
                    merges=merges[: 3 * inf["n_split"]].reshape(-1, 3),
                    win_row=self.window_rows())

    def close(self):
        if self._h is not None:
            load_library().f3s_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()


def run(plan, Q, K, V, scale=None, out=None, stream=None):
    """O = softmax_rows(mask_A(scale Q K^T)) V through f3s_run / f3s_run_mh.

    Q, K, V: fp16 device tensors [N, d] (one head) or [N, H, d] (H heads
    sharing the plan); out: optional fp32 tensor of the same shape; the call
    is asynchronous on ``stream`` (default: torch's current stream).
    """
    L = load_library()
    shape = tuple(Q.shape)
    for t, n in ((Q, "Q"), (K, "K"), (V, "V")):
        _check_device_tensor(t, n, torch.float16, plan.device)
        if t.dim() not in (2, 3) or t.shape[0] != plan.N:
            raise ValueError(f"{n} must be [N, d] or [N, H, d] with N = {plan.N}")
        if tuple(t.shape) != shape:
            raise ValueError("Q, K, V must share one shape")
    H = shape[1] if len(shape) == 3 else 1
    d = shape[-1]
    if out is None:
        out = torch.empty(shape, dtype=torch.float32, device=Q.device)
    else:
        _check_device_tensor(out, "out", torch.float32, Q.device)
        if tuple(out.shape) != shape:
            raise ValueError("out must have the shape of Q")
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    if stream is None:
        stream = torch.cuda.current_stream(Q.device)
    rc = L.f3s_run_mh(plan.handle, Q.data_ptr(), K.data_ptr(), V.data_ptr(),
                      out.data_ptr(), int(H), int(d), float(scale),
                      ctypes.c_void_p(stream.cuda_stream))
    if rc != F3S_OK:
        raise F3SError(rc, "f3s_run_mh")
    return out


def forward(plan, Q, K, V, scale=None, out=None, lse=None, stream=None):
    """f3s_forward: returns (O, lse) with lse fp32 [N] or [N, H]."""
    shape = _qkv_shape(Q)
    H = shape[1] if len(shape) == 3 else 1
    for t, n in ((Q, "Q"), (K, "K"), (V, "V")):
        _check_device_tensor(t, n, torch.float16, plan.device)
        if tuple(t.shape) != shape or shape[0] != plan.N:
            raise ValueError("Q, K, V must share one [N, d] / [N, H, d] shape")
    if lse is None:
        lse = torch.empty(shape[:-1], dtype=torch.float32, device=Q.device)
    _check_device_tensor(lse, "lse", torch.float32, Q.device)
    if lse.numel() != plan.N * H:
        raise ValueError("lse must hold N * H values")
    if out is None:
        out = torch.empty(shape, dtype=torch.float32, device=Q.device)
    _check_device_tensor(out, "out", torch.float32, Q.device)
    if tuple(out.shape) != shape:
        raise ValueError("out must have the shape of Q")
    d = shape[-1]
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    if stream is None:
        stream = torch.cuda.current_stream(Q.device)
    rc = load_library().f3s_forward(plan.handle, Q.data_ptr(), K.data_ptr(), V.data_ptr(),
                                    out.data_ptr(), lse.data_ptr(), int(H), int(d),
                                    float(scale), ctypes.c_void_p(stream.cuda_stream))
    if rc != F3S_OK:
        raise F3SError(rc, "f3s_forward")
    return out, lse


# f3s_dtype_t codes
_DTYPE_CODE = {torch.float16: 0, torch.bfloat16: 1, torch.float32: 2,
               torch.float8_e4m3fn: 3}


def forward_typed(plan, Q, K, V, out_dtype=torch.float32, scale=None, out=None,
                  lse=None, want_lse=False, stream=None):
    """f3s_forward_typed: Q, K, V fp16, bf16 or float8_e4m3fn ([N, d] or
    [N, H, d]); O of ``out_dtype`` (fp32 or fp16).  Returns (O, lse) with lse
    None unless ``want_lse`` or an ``lse`` tensor is given."""
    shape = _qkv_shape(Q)
    H = shape[1] if len(shape) == 3 else 1
    if Q.dtype not in (torch.float16, torch.bfloat16, torch.float8_e4m3fn):
        raise TypeError(f"Q must be float16, bfloat16 or float8_e4m3fn, got {Q.dtype}")
    for t, n in ((Q, "Q"), (K, "K"), (V, "V")):
        _check_device_tensor(t, n, Q.dtype, plan.device)
        if tuple(t.shape) != shape or shape[0] != plan.N:
            raise ValueError("Q, K, V must share one [N, d] / [N, H, d] shape")
    if out is None:
        out = torch.empty(shape, dtype=out_dtype, device=Q.device)
    _check_device_tensor(out, "out", out_dtype, Q.device)
    if tuple(out.shape) != shape:
        raise ValueError("out must have the shape of Q")
    if lse is None and want_lse:
        lse = torch.empty(shape[:-1], dtype=torch.float32, device=Q.device)
    if lse is not None:
        _check_device_tensor(lse, "lse", torch.float32, Q.device)
        if lse.numel() != plan.N * H:
            raise ValueError("lse must hold N * H values")
    d = shape[-1]
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    if stream is None:
        stream = torch.cuda.current_stream(Q.device)
    rc = load_library().f3s_forward_typed(
        plan.handle, Q.data_ptr(), K.data_ptr(), V.data_ptr(), _DTYPE_CODE[Q.dtype],
        out.data_ptr(), _DTYPE_CODE.get(out_dtype, -1),
        lse.data_ptr() if lse is not None else None, int(H), int(d), float(scale),
        ctypes.c_void_p(stream.cuda_stream))
    if rc != F3S_OK:
        raise F3SError(rc, "f3s_forward_typed")
    return out, lse


def backward(plan, plan_t, Q, K, V, O, dO, lse, scale=None, stream=None):
    """f3s_backward_typed: returns (dQ, dK, dV) fp32 for fp16 or bf16 Q, K, V,
    dO (the per-row (lse, delta) records it needs go to a buffer allocated
    here)."""
    shape = _qkv_shape(Q)
    H = shape[1] if len(shape) == 3 else 1
    d = shape[-1]
    if Q.dtype not in (torch.float16, torch.bfloat16):
        raise TypeError("Q, K, V, dO must be float16 or bfloat16")
    for t, n in ((Q, "Q"), (K, "K"), (V, "V"), (dO, "dO")):
        _check_device_tensor(t, n, Q.dtype, plan.device)
        if tuple(t.shape) != shape or shape[0] != plan.N:
            raise ValueError(f"{n} must have the shape of Q, with N = {plan.N} rows")
    _check_device_tensor(O, "O", torch.float32, Q.device)
    _check_device_tensor(lse, "lse", torch.float32, Q.device)
    if tuple(O.shape) != shape or lse.numel() != plan.N * H:
        raise ValueError("O must match Q; lse must hold N * H values")
    dQ, dK, dV = (torch.empty(shape, dtype=torch.float32, device=Q.device) for _ in range(3))
    row_stats = torch.empty(shape[:-1] + (2,), dtype=torch.float32, device=Q.device)
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    if stream is None:
        stream = torch.cuda.current_stream(Q.device)
    rc = load_library().f3s_backward_typed(
        plan.handle, plan_t.handle, Q.data_ptr(), K.data_ptr(), V.data_ptr(),
        _DTYPE_CODE[Q.dtype], O.data_ptr(), dO.data_ptr(), lse.data_ptr(),
        row_stats.data_ptr(), dQ.data_ptr(), dK.data_ptr(), dV.data_ptr(), int(H), int(d),
        float(scale), ctypes.c_void_p(stream.cuda_stream))
    if rc != F3S_OK:
        raise F3SError(rc, "f3s_backward_typed")
    return dQ, dK, dV


def run_raw(plan, q_ptr, k_ptr, v_ptr, o_ptr, d, scale, stream_handle):
    """f3s_run on raw device addresses (returns the status code)."""
    return load_library().f3s_run(plan.handle, q_ptr, k_ptr, v_ptr, o_ptr, int(d),
                                  float(scale), ctypes.c_void_p(stream_handle))


def probe_stream(kind, buf, out=None, stream=None):
    """One streaming probe over the bytes of device tensor ``buf``:
    kind "read" (out: a uint32 device tensor of >= 256 elements, the
    never-written sink), "copy" (out: a tensor of buf's size) or "write"."""
    L = load_library()
    if not isinstance(buf, torch.Tensor) or not buf.is_cuda or not buf.is_contiguous():
        raise TypeError("buf must be a contiguous device tensor")
    nbytes = buf.numel() * buf.element_size()
    if stream is None:
        stream = torch.cuda.current_stream(buf.device)
    s = ctypes.c_void_p(stream.cuda_stream)
    if kind == "read":
        if out is None or out.numel() * out.element_size() < 1024 or out.device != buf.device:
            raise ValueError("read needs a sink of at least 1 KiB on buf's device")
        rc = L.f3s_probe_read(buf.data_ptr(), nbytes, out.data_ptr(), s)
    elif kind == "copy":
        if (out is None or out.numel() * out.element_size() != nbytes
                or out.device != buf.device or not out.is_contiguous()):
            raise ValueError("copy needs a contiguous destination of buf's size and device")
        rc = L.f3s_probe_copy(buf.data_ptr(), out.data_ptr(), nbytes, s)
    elif kind == "write":
        rc = L.f3s_probe_write(buf.data_ptr(), nbytes, 0x5A5A5A5A, s)
    else:
        raise ValueError(f"unknown probe {kind}")
    if rc != F3S_OK:
        raise F3SError(rc, f"f3s_probe_{kind}")


def probe_gather(plan, Q, K, V, out, stream=None, lds=False):
    """f3s_probe_gather: the fused kernel's memory accesses on ``plan`` for
    fp16 Q, K, V [N, d] and fp32 out [N, d], without its arithmetic
    (``lds``: f3s_probe_gather_lds, the K and V rows loaded into LDS with no
    limit on the rows in flight)."""
    shape = tuple(Q.shape)
    for t, n in ((Q, "Q"), (K, "K"), (V, "V")):
        _check_device_tensor(t, n, torch.float16, plan.device)
        if t.dim() != 2 or tuple(t.shape) != shape or shape[0] != plan.N:
            raise ValueError("Q, K, V must be [N, d]")
    _check_device_tensor(out, "out", torch.float32, plan.device)
    if tuple(out.shape) != shape:
        raise ValueError("out must have the shape of Q")
    if stream is None:
        stream = torch.cuda.current_stream(Q.device)
    L = load_library()
    fn = L.f3s_probe_gather_lds if lds else L.f3s_probe_gather
    rc = fn(plan.handle, Q.data_ptr(), K.data_ptr(), V.data_ptr(), out.data_ptr(),
            int(shape[1]), ctypes.c_void_p(stream.cuda_stream))
    if rc != F3S_OK:
        raise F3SError(rc, "f3s_probe_gather_lds" if lds else "f3s_probe_gather")


def probe_rows(table, rows, row_bytes, sink, in_flight=8, workgroups=2048, rounds=4,
               stream=None):
    """f3s_probe_rows: random gathers of whole rows of ``row_bytes`` bytes
    from the first ``rows`` rows of device tensor ``table``, ``in_flight``
    rows in flight per thread; returns the bytes one call reads
    (workgroups * rounds * in_flight * 4096)."""
    if not isinstance(table, torch.Tensor) or not table.is_cuda or not table.is_contiguous():
        raise TypeError("table must be a contiguous device tensor")
    if int(rows) * int(row_bytes) > table.numel() * table.element_size():
        raise ValueError("rows * row_bytes exceeds the table")
    if (sink is None or sink.device != table.device
            or sink.numel() * sink.element_size() < 1024):
        raise ValueError("sink must hold 256 uint32 on the table's device")
    if stream is None:
        stream = torch.cuda.current_stream(table.device)
    rc = load_library().f3s_probe_rows(table.data_ptr(), int(rows), int(row_bytes),
                                       int(in_flight), int(workgroups), int(rounds),
                                       sink.data_ptr(), ctypes.c_void_p(stream.cuda_stream))
    if rc != F3S_OK:
        raise F3SError(rc, "f3s_probe_rows")
    return int(workgroups) * int(rounds) * int(in_flight) * 4096


def run_trace(plan, Q, K, V, scale=None, out=None, stream=None):
    """f3s_run_trace: one-head fp16 -> fp32 forward (O as f3s_run) plus one
    record per workgroup (start, end, compute unit); returns (O, records)
    with records a uint32 device tensor [n_items, 8]."""
    shape = tuple(Q.shape)
    for t, n in ((Q, "Q"), (K, "K"), (V, "V")):
        _check_device_tensor(t, n, torch.float16, plan.device)
        if t.dim() != 2 or tuple(t.shape) != shape or shape[0] != plan.N:
            raise ValueError("Q, K, V must be [N, d]")
    if out is None:
        out = torch.empty(shape, dtype=torch.float32, device=Q.device)
    _check_device_tensor(out, "out", torch.float32, plan.device)
    if tuple(out.shape) != shape:
        raise ValueError("out must have the shape of Q")
    n = max(1, plan.info["n_items"])
    rec = torch.zeros((n, 8), dtype=torch.int32, device=Q.device)
    d = shape[1]
    if scale is None:
        scale = 1.0 / math.sqrt(d)
    if stream is None:
        stream = torch.cuda.current_stream(Q.device)
    rc = load_library().f3s_run_trace(plan.handle, Q.data_ptr(), K.data_ptr(), V.data_ptr(),
                                      out.data_ptr(), int(d), float(scale), rec.data_ptr(),
                                      rec.numel() * 4, ctypes.c_void_p(stream.cuda_stream))
    if rc != F3S_OK:
        raise F3SError(rc, "f3s_run_trace")
    return out, rec


def wall_clock_khz(device=0):
    """Frequency of the trace records' clock (kHz)."""
    return int(load_library().f3s_wall_clock_khz(int(device)))
