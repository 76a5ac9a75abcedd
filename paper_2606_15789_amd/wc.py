"""Python binding of libwc (ctypes): argument marshalling only.

Every step of the decode runs in libwc's HIP kernel; this module converts
numpy / torch objects to the plain pointers and sizes of the C ABI declared in
``include/wc.h`` and raises on any non-zero status.  There is no fallback: if
``libwc.so`` is missing or fails to load, every call raises.
"""

from __future__ import annotations

import ctypes as C
import os

import numpy as np

from . import build as _build

DTYPES = {"bf16": 1, "fp16": 2, "u8": 3, "u4": 4, "fp8_e4m3": 5, "fp8_e5m2": 6, "fp4_e2m1": 7}
STATUS = {0: "WC_OK", -1: "WC_EINVAL", -2: "WC_ENOMEM", -3: "WC_ECORRUPT", -4: "WC_EHIP",
          -5: "WC_EUNSUPPORTED"}
DERR = {1: "WC_DERR_INDEX", 2: "WC_DERR_STATE", 4: "WC_DERR_CURSOR", 8: "WC_DERR_TABLE"}

# Every function the header declares; the library must export all of them.
EXPORTS = ["wc_analyze", "wc_encode", "wc_open", "wc_decode", "wc_gemv", "wc_free",
           "wc_version", "wc_analyze_device", "wc_encode_device_bounds", "wc_encode_device",
           "wc_gemm_workspace_bytes", "wc_gemm", "wc_gemm_i8", "wc_gemv_mx", "wc_gemv_w4",
           "wc_stream", "wc_analyze_device_static"]

ANALYZE_WORKSPACE_BYTES = 524288  # WC_ANALYZE_WORKSPACE_BYTES


class WcError(RuntimeError):
    def __init__(self, what, rc):
        super().__init__(f"{what} failed: {STATUS.get(rc, rc)}")
        self.rc = rc


class _Tensor(C.Structure):
    _fields_ = [("host_ptr", C.c_void_p), ("nbytes", C.c_uint64), ("dtype", C.c_int32),
                ("reserved", C.c_int32), ("rows", C.c_uint64), ("cols", C.c_uint64)]


class _Params(C.Structure):
    _fields_ = [("chunk_bytes", C.c_uint32), ("lanes", C.c_uint32), ("prob_bits", C.c_uint32),
                ("n_threads", C.c_uint32), ("tile_rows", C.c_uint32), ("tile_cols", C.c_uint32),
                ("codebook", C.c_uint32), ("tile_order", C.c_uint32)]


CODEBOOKS = {"tensor": 0, "layer": 1}


class _Stats(C.Structure):
    _fields_ = [("n_fields", C.c_uint32), ("alphabet", C.c_uint32 * 2),
                ("count", C.c_uint64 * 2), ("hist", (C.c_uint64 * 256) * 2),
                ("H", C.c_double * 2), ("H_joint16", C.c_double),
                ("bound_bytes", C.c_double), ("bound_bytes_raw8", C.c_double)]


class _Blob(C.Structure):
    _fields_ = [("data", C.POINTER(C.c_uint8)), ("size", C.c_uint64),
                ("n_tensors", C.c_uint32), ("reserved", C.c_uint32),
                ("n_chunks", C.c_uint64), ("out_bytes", C.POINTER(C.c_uint64)),
                ("meta_bytes", C.c_uint64), ("record_hdr_bytes", C.c_uint64),
                ("state_bytes", C.c_uint64), ("word_bytes", C.c_uint64),
                ("pad_bytes", C.c_uint64), ("raw_bytes", C.c_uint64),
                ("priv", C.c_void_p)]


_lib = None


def lib():
    """Load libwc.so (building it first only if nothing is built)."""
    global _lib
    if _lib is None:
        # WC_LIB selects another build of libwc (for A/B measurements of kernel variants)
        path = os.environ.get("WC_LIB") or _build.ensure_built()
        L = C.CDLL(path)
        L.wc_analyze.argtypes = [C.POINTER(_Tensor), C.POINTER(_Stats)]
        L.wc_analyze.restype = C.c_int
        L.wc_encode.argtypes = [C.POINTER(_Tensor), C.c_uint32, C.POINTER(_Params),
                                C.POINTER(C.POINTER(_Blob))]
        L.wc_encode.restype = C.c_int
        L.wc_open.argtypes = [C.c_void_p, C.c_uint64, C.POINTER(C.POINTER(_Blob))]
        L.wc_open.restype = C.c_int
        L.wc_decode.argtypes = [C.POINTER(_Blob), C.c_void_p, C.POINTER(C.c_void_p), C.c_uint32,
                                C.c_void_p, C.c_void_p]
        L.wc_decode.restype = C.c_int
        L.wc_gemv.argtypes = [C.POINTER(_Blob), C.c_void_p, C.c_uint32,
                              C.POINTER(C.c_uint32), C.POINTER(C.c_void_p), C.c_uint32,
                              C.POINTER(C.c_void_p), C.c_void_p, C.c_void_p]
        L.wc_gemv.restype = C.c_int
        L.wc_gemm_workspace_bytes.argtypes = [C.POINTER(_Blob), C.c_uint32,
                                              C.POINTER(C.c_uint32), C.POINTER(C.c_void_p),
                                              C.c_uint32, C.POINTER(C.c_uint64)]
        L.wc_gemm_workspace_bytes.restype = C.c_int
        L.wc_gemm.argtypes = [C.POINTER(_Blob), C.c_void_p, C.c_uint32, C.POINTER(C.c_uint32),
                              C.POINTER(C.c_void_p), C.c_uint32, C.POINTER(C.c_void_p),
                              C.c_void_p, C.c_uint64, C.c_void_p, C.c_void_p]
        L.wc_gemm.restype = C.c_int
        L.wc_gemm_i8.argtypes = [C.POINTER(_Blob), C.c_void_p, C.c_uint32, C.POINTER(C.c_uint32),
                                 C.POINTER(C.c_void_p), C.c_uint32, C.POINTER(C.c_void_p),
                                 C.c_void_p, C.c_void_p]
        L.wc_gemm_i8.restype = C.c_int
        L.wc_gemv_mx.argtypes = [C.POINTER(_Blob), C.c_void_p, C.c_uint32, C.POINTER(C.c_uint32),
                                 C.POINTER(C.c_void_p), C.POINTER(C.c_void_p), C.c_uint32,
                                 C.POINTER(C.c_void_p), C.c_void_p, C.c_void_p]
        L.wc_gemv_mx.restype = C.c_int
        L.wc_gemv_w4.argtypes = [C.POINTER(_Blob), C.c_void_p, C.c_uint32, C.POINTER(C.c_uint32),
                                 C.POINTER(C.c_void_p), C.POINTER(C.c_void_p),
                                 C.POINTER(C.c_void_p), C.c_uint32, C.POINTER(C.c_void_p),
                                 C.c_void_p, C.c_void_p]
        L.wc_gemv_w4.restype = C.c_int
        L.wc_analyze_device.argtypes = [C.POINTER(_Tensor), C.c_void_p, C.c_uint64, C.c_void_p,
                                        C.POINTER(_Stats)]
        L.wc_analyze_device.restype = C.c_int
        L.wc_analyze_device_static.argtypes = [C.POINTER(_Tensor), C.c_void_p, C.POINTER(_Stats)]
        L.wc_analyze_device_static.restype = C.c_int
        L.wc_encode_device_bounds.argtypes = [C.POINTER(_Tensor), C.c_uint32, C.POINTER(_Params),
                                              C.POINTER(C.c_uint64), C.POINTER(C.c_uint64)]
        L.wc_encode_device_bounds.restype = C.c_int
        L.wc_encode_device.argtypes = [C.POINTER(_Tensor), C.c_uint32, C.POINTER(_Params),
                                       C.c_void_p, C.c_uint64, C.c_void_p, C.c_uint64,
                                       C.c_void_p, C.c_void_p]
        L.wc_encode_device.restype = C.c_int
        L.wc_stream.argtypes = [C.c_void_p, C.c_uint64, C.c_void_p, C.c_uint64, C.c_uint32,
                                C.c_void_p, C.POINTER(C.c_uint64)]
        L.wc_stream.restype = C.c_int
        L.wc_free.argtypes = [C.POINTER(_Blob)]
        L.wc_free.restype = None
        L.wc_version.restype = C.c_int32
        _lib = L
    return _lib


def library_path() -> str:
    return os.environ.get("WC_LIB") or _build.LIB


def _bytes(data) -> np.ndarray:
    a = np.ascontiguousarray(data)
    return a.view(np.uint8).reshape(-1)


def analyze(dtype: str, data) -> dict:
    """wc_analyze: per-field histograms and empirical entropy of one tensor."""
    b = _bytes(data)
    t = _Tensor(b.ctypes.data if b.size else None, b.size, DTYPES[dtype], 0, 0, 0)
    st = _Stats()
    rc = lib().wc_analyze(C.byref(t), C.byref(st))
    if rc:
        raise WcError("wc_analyze", rc)
    return _stats_dict(st)


def _stats_dict(st) -> dict:
    nf = st.n_fields
    return {"n_fields": nf, "alphabet": [st.alphabet[i] for i in range(nf)],
            "count": [st.count[i] for i in range(nf)],
            "hist": [np.array(st.hist[i][:st.alphabet[i]], np.uint64) for i in range(nf)],
            "H": [st.H[i] for i in range(nf)], "H_joint16": st.H_joint16,
            "bound_bytes": st.bound_bytes, "bound_bytes_raw8": st.bound_bytes_raw8}


class Blob:
    """Owner of a wc_blob (released with wc_free)."""

    def __init__(self, ptr):
        self._p = ptr
        b = ptr.contents
        self.size = int(b.size)
        self.n_tensors = int(b.n_tensors)
        self.n_chunks = int(b.n_chunks)
        self.out_bytes = [int(b.out_bytes[i]) for i in range(self.n_tensors)]
        self.breakdown = {k: int(getattr(b, k)) for k in
                          ("meta_bytes", "record_hdr_bytes", "state_bytes", "word_bytes",
                           "pad_bytes", "raw_bytes")}

    @property
    def ptr(self):
        if self._p is None:
            raise ValueError("blob already freed")
        return self._p

    def array(self) -> np.ndarray:
        """Zero-copy numpy view of the host blob bytes (valid until free)."""
        b = self.ptr.contents
        return np.ctypeslib.as_array(b.data, shape=(self.size,))

    def tobytes(self) -> bytes:
        return C.string_at(self.ptr.contents.data, self.size)

    def shape(self, t: int):
        """(rows, cols) of tensor t in symbol elements, from its descriptor in
        the blob header (blob format: 64-byte header, 96-byte descriptors with
        rows and cols at bytes 64 and 72); (0, 0) for an unshaped tensor."""
        d = np.frombuffer(self.array()[64 + 96 * t: 64 + 96 * (t + 1)].tobytes(), np.uint64)
        return int(d[8]), int(d[9])

    def dtype(self, t: int) -> str:
        """Storage format of tensor t (the descriptor's first u32)."""
        code = int(np.frombuffer(self.array()[64 + 96 * t: 64 + 96 * t + 4].tobytes(), np.uint32)[0])
        return {v: k for k, v in DTYPES.items()}[code]

    def payload_bytes(self) -> int:
        """Lane states + words + raw bytes (what the entropy bound is compared with)."""
        d = self.breakdown
        return d["state_bytes"] + d["word_bytes"] + d["raw_bytes"]

    def free(self):
        if self._p is not None:
            lib().wc_free(self._p)
            self._p = None

    def __del__(self):
        try:
            self.free()
        except Exception:
            pass


def encode(tensors, chunk_bytes: int = 65536, lanes: int = 64, threads: int = 0, tile=(0, 0),
           codebook: str = "tensor", tile_order: int = 0) -> Blob:
    """wc_encode of a list of (dtype, host array[, (rows, cols)]) entries.

    The shape is in symbol elements (16-bit words, bytes or nibbles); `tile`
    = (tile_rows, tile_cols) cuts every tensor it divides into one chunk per
    tile (tile_order 0: row-major tiles, 1: column blocks, the wc_gemv layout).
    codebook "layer" shares one table among the tensors of a dtype.
    """
    keep = [_bytes(e[1]) for e in tensors]
    arr = (_Tensor * len(tensors))()
    for i, (e, b) in enumerate(zip(tensors, keep)):
        rows, cols = e[2] if len(e) > 2 and e[2] is not None else (0, 0)
        arr[i] = _Tensor(b.ctypes.data if b.size else None, b.size, DTYPES[e[0]], 0, rows, cols)
    prm = _Params(chunk_bytes, lanes, 12, threads, tile[0], tile[1], CODEBOOKS[codebook],
                  tile_order)
    out = C.POINTER(_Blob)()
    rc = lib().wc_encode(arr, len(tensors), C.byref(prm), C.byref(out))
    if rc:
        raise WcError("wc_encode", rc)
    return Blob(out)


def open_blob(data) -> Blob:
    """wc_open: validate and take a copy of blob bytes made elsewhere."""
    b = _bytes(np.frombuffer(data, np.uint8) if isinstance(data, (bytes, bytearray)) else data)
    out = C.POINTER(_Blob)()
    rc = lib().wc_open(b.ctypes.data, b.size, C.byref(out))
    if rc:
        raise WcError("wc_open", rc)
    return Blob(out)


def decode(blob: Blob, dev_blob: int, dev_dst, stream: int = 0, dev_err: int = 0) -> None:
    """wc_decode with raw device pointers (ints); asynchronous on `stream`."""
    ptrs = (C.c_void_p * max(1, len(dev_dst)))(*[p or None for p in dev_dst])
    rc = lib().wc_decode(blob.ptr, C.c_void_p(dev_blob), ptrs, len(dev_dst),
                         C.c_void_p(stream or None), C.c_void_p(dev_err or None))
    if rc:
        raise WcError("wc_decode", rc)


def gemv(blob: Blob, dev_blob: int, tensors, dev_x, m: int, dev_y, stream: int = 0,
         dev_err: int = 0) -> None:
    """wc_gemv with raw device pointers: y_i (m x N fp32) += x_i (m x K bf16) * W_i^T for
    each job i (tensors, dev_x, dev_y: equal-length lists), in one launch."""
    n = len(tensors)
    ts = (C.c_uint32 * max(n, 1))(*tensors)
    xs = (C.c_void_p * max(n, 1))(*[p or None for p in dev_x])
    ys = (C.c_void_p * max(n, 1))(*[p or None for p in dev_y])
    rc = lib().wc_gemv(blob.ptr, C.c_void_p(dev_blob), n, ts, xs, m, ys,
                       C.c_void_p(stream or None), C.c_void_p(dev_err or None))
    if rc:
        raise WcError("wc_gemv", rc)


def gemm_workspace_bytes(blob: Blob, tensors, dev_x, m: int) -> int:
    """wc_gemm_workspace_bytes: device bytes wc_gemm needs for these jobs (0 up
    to 64 rows of x; jobs with the same x share its packed copy)."""
    n = len(tensors)
    ts = (C.c_uint32 * max(n, 1))(*tensors)
    xs = (C.c_void_p * max(n, 1))(*[p or None for p in dev_x])
    out = C.c_uint64(0)
    rc = lib().wc_gemm_workspace_bytes(blob.ptr, n, ts, xs, m, C.byref(out))
    if rc:
        raise WcError("wc_gemm_workspace_bytes", rc)
    return out.value


def gemm(blob: Blob, dev_blob: int, tensors, dev_x, m: int, dev_y, workspace: int = 0,
         workspace_bytes: int = 0, stream: int = 0, dev_err: int = 0) -> None:
    """wc_gemm with raw device pointers: wc_gemv for up to 64 rows of x, the
    shared fused GEMM (packed x in the caller's workspace) above."""
    n = len(tensors)
    ts = (C.c_uint32 * max(n, 1))(*tensors)
    xs = (C.c_void_p * max(n, 1))(*[p or None for p in dev_x])
    ys = (C.c_void_p * max(n, 1))(*[p or None for p in dev_y])
    rc = lib().wc_gemm(blob.ptr, C.c_void_p(dev_blob), n, ts, xs, m, ys,
                       C.c_void_p(workspace or None), workspace_bytes,
                       C.c_void_p(stream or None), C.c_void_p(dev_err or None))
    if rc:
        raise WcError("wc_gemm", rc)


def gemm_i8(blob: Blob, dev_blob: int, tensors, dev_x, m: int, dev_y, stream: int = 0,
            dev_err: int = 0) -> None:
    """wc_gemm_i8 with raw device pointers: y_i (m x N int32) += x_i (m x K int8)
    * W_i^T (int8), exactly, in one launch."""
    n = len(tensors)
    ts = (C.c_uint32 * max(n, 1))(*tensors)
    xs = (C.c_void_p * max(n, 1))(*[p or None for p in dev_x])
    ys = (C.c_void_p * max(n, 1))(*[p or None for p in dev_y])
    rc = lib().wc_gemm_i8(blob.ptr, C.c_void_p(dev_blob), n, ts, xs, m, ys,
                          C.c_void_p(stream or None), C.c_void_p(dev_err or None))
    if rc:
        raise WcError("wc_gemm_i8", rc)


def gemv_mx(blob: Blob, dev_blob: int, tensors, dev_scales, dev_x, m: int, dev_y,
            stream: int = 0, dev_err: int = 0) -> None:
    """wc_gemv_mx with raw device pointers: y_i (m x N float) += x_i (m x K bf16)
    * W_i^T for MXFP4 W_i (e2m1 codes in the blob, e8m0 scales at dev_scales[i])."""
    n = len(tensors)
    ts = (C.c_uint32 * max(n, 1))(*tensors)
    ss = (C.c_void_p * max(n, 1))(*[p or None for p in dev_scales])
    xs = (C.c_void_p * max(n, 1))(*[p or None for p in dev_x])
    ys = (C.c_void_p * max(n, 1))(*[p or None for p in dev_y])
    rc = lib().wc_gemv_mx(blob.ptr, C.c_void_p(dev_blob), n, ts, ss, xs, m, ys,
                          C.c_void_p(stream or None), C.c_void_p(dev_err or None))
    if rc:
        raise WcError("wc_gemv_mx", rc)


def gemv_w4(blob: Blob, dev_blob: int, tensors, dev_scales, dev_zeros, dev_x, m: int, dev_y,
            stream: int = 0, dev_err: int = 0) -> None:
    """wc_gemv_w4 with raw device pointers: y_i += x_i * W_i^T for int4 W_i (packed
    codes as the blob's byte tensor, fp16 scales per 128 at dev_scales[i], zero
    points at dev_zeros[i] or 0 for two's-complement codes; dev_zeros None: all
    two's-complement)."""
    n = len(tensors)
    ts = (C.c_uint32 * max(n, 1))(*tensors)
    ss = (C.c_void_p * max(n, 1))(*[p or None for p in dev_scales])
    zs = None if dev_zeros is None else (C.c_void_p * max(n, 1))(*[p or None for p in dev_zeros])
    xs = (C.c_void_p * max(n, 1))(*[p or None for p in dev_x])
    ys = (C.c_void_p * max(n, 1))(*[p or None for p in dev_y])
    rc = lib().wc_gemv_w4(blob.ptr, C.c_void_p(dev_blob), n, ts, ss, zs, xs, m, ys,
                          C.c_void_p(stream or None), C.c_void_p(dev_err or None))
    if rc:
        raise WcError("wc_gemv_w4", rc)


def stream_bytes(dev_src: int, src_bytes: int, dev_dst: int, dst_bytes: int, blocks: int = 0,
                 stream: int = 0) -> int:
    """wc_stream (a measuring aid, no decoding): read src_bytes once and write
    dst_bytes once, non-temporal, on `stream`; returns the bytes it reads."""
    rd = C.c_uint64(0)
    rc = lib().wc_stream(C.c_void_p(dev_src or None), src_bytes, C.c_void_p(dev_dst or None),
                         dst_bytes, blocks, C.c_void_p(stream or None), C.byref(rd))
    if rc:
        raise WcError("wc_stream", rc)
    return rd.value


# --- torch plumbing: device memory and streams only ---------------------------

def to_device(blob: Blob, device="cuda"):
    """Copy the blob bytes into a new uint8 device tensor."""
    import torch
    host = torch.from_numpy(blob.array())
    return host.to(device)


def decode_torch(blob: Blob, dev_blob, outs=None, stream=None, err=None):
    """Decode into uint8 device tensors (allocated if `outs` is None).

    Returns the list of output tensors.  `err` (int32 device tensor of one
    element) receives the WC_DERR_* bits; the caller reads it after syncing.
    """
    import torch
    dev = dev_blob.device
    if outs is None:
        outs = [torch.empty(n, dtype=torch.uint8, device=dev) for n in blob.out_bytes]
    for o, n in zip(outs, blob.out_bytes):
        if o.numel() * o.element_size() < n or not o.is_contiguous():
            raise ValueError("output tensor too small or not contiguous")
    if stream is None:
        stream = torch.cuda.current_stream(dev)
    decode(blob, dev_blob.data_ptr(), [o.data_ptr() if n else 0 for o, n in zip(outs, blob.out_bytes)],
           stream.cuda_stream, err.data_ptr() if err is not None else 0)
    return outs


def describe_errors(bits: int) -> list:
    return [name for b, name in DERR.items() if bits & b]


def gemv_torch(blob: Blob, dev_blob, tensors, xs, ys=None, stream=None, err=None):
    """Fused decode-GEMM into float32 tensors, one launch: ys[i] += xs[i] @ W_i^T for
    W_i = tensor tensors[i] (ys zeroed and returned if None)."""
    import torch
    m = xs[0].shape[0]
    for x in xs:
        if x.dtype != torch.bfloat16 or not x.is_contiguous() or x.shape[0] != m:
            raise ValueError("xs must be contiguous bfloat16 tensors with equal row counts")
    if ys is None:
        ys = [torch.zeros((m, blob.shape(t)[0]), dtype=torch.float32, device=x.device)
              for t, x in zip(tensors, xs)]
    if stream is None:
        stream = torch.cuda.current_stream(xs[0].device)
    gemv(blob, dev_blob.data_ptr(), list(tensors), [x.data_ptr() for x in xs], m,
         [y.data_ptr() for y in ys], stream.cuda_stream, err.data_ptr() if err is not None else 0)
    return ys


# --- device-side analysis and encoder ----------------------------------------
# wc_dtensor has wc_tensor's layout, with a device pointer in the first field.

def _dtensors(entries):
    """ctypes wc_dtensor array of (dtype, device tensor[, (rows, cols)]) entries."""
    arr = (_Tensor * len(entries))()
    for i, e in enumerate(entries):
        x = e[1]
        if not x.is_contiguous():
            raise ValueError("device tensors must be contiguous")
        nbytes = x.numel() * x.element_size()
        rows, cols = e[2] if len(e) > 2 and e[2] is not None else (0, 0)
        arr[i] = _Tensor(x.data_ptr() if nbytes else None, nbytes, DTYPES[e[0]], 0, rows, cols)
    return arr


def _params(chunk_bytes, lanes, tile, codebook, tile_order):
    return _Params(chunk_bytes, lanes, 12, 0, tile[0], tile[1], CODEBOOKS[codebook], tile_order)


def analyze_device(dtype: str, x, workspace=None, stream=None) -> dict:
    """wc_analyze_device of a device tensor (synchronises `stream`)."""
    import torch
    t = _dtensors([(dtype, x)])
    if workspace is None:
        workspace = torch.empty(ANALYZE_WORKSPACE_BYTES, dtype=torch.uint8, device=x.device)
    if stream is None:
        stream = torch.cuda.current_stream(x.device)
    st = _Stats()
    rc = lib().wc_analyze_device(t, C.c_void_p(workspace.data_ptr()), workspace.numel(),
                                 C.c_void_p(stream.cuda_stream or None), C.byref(st))
    if rc:
        raise WcError("wc_analyze_device", rc)
    return _stats_dict(st)


def analyze_device_static(dtype: str, x, stream=None) -> dict:
    """wc_analyze_device_static of a tensor on the current device: no workspace,
    the bins are the library's own device array (synchronises `stream`)."""
    import torch
    t = _dtensors([(dtype, x)])
    if stream is None:
        stream = torch.cuda.current_stream(x.device)
    st = _Stats()
    rc = lib().wc_analyze_device_static(t, C.c_void_p(stream.cuda_stream or None), C.byref(st))
    if rc:
        raise WcError("wc_analyze_device_static", rc)
    return _stats_dict(st)


def encode_device_bounds(entries, chunk_bytes: int = 65536, lanes: int = 64, tile=(0, 0),
                         codebook: str = "tensor", tile_order: int = 0):
    """(blob capacity, workspace bytes) wc_encode_device needs.  `entries` are
    (dtype, nbytes[, (rows, cols)]) or (dtype, tensor[, shape]) entries."""
    arr = (_Tensor * len(entries))()
    for i, e in enumerate(entries):
        nb = e[1] if isinstance(e[1], int) else e[1].numel() * e[1].element_size()
        rows, cols = e[2] if len(e) > 2 and e[2] is not None else (0, 0)
        arr[i] = _Tensor(None, nb, DTYPES[e[0]], 0, rows, cols)
    prm = _params(chunk_bytes, lanes, tile, codebook, tile_order)
    cap, ws = C.c_uint64(), C.c_uint64()
    rc = lib().wc_encode_device_bounds(arr, len(entries), C.byref(prm), C.byref(cap), C.byref(ws))
    if rc:
        raise WcError("wc_encode_device_bounds", rc)
    return cap.value, ws.value


def encode_device(entries, chunk_bytes: int = 65536, lanes: int = 64, tile=(0, 0),
                  codebook: str = "tensor", tile_order: int = 0, blob=None, workspace=None,
                  size=None, stream=None):
    """wc_encode_device of (dtype, device tensor[, (rows, cols)]) entries.

    Returns (blob, size): a uint8 device tensor of the capacity the bounds
    give and an int64 device tensor of one element that receives the blob's
    size; both are valid after `stream` (default: the current one) syncs.
    """
    import torch
    dev = entries[0][1].device
    cap, wsb = encode_device_bounds([(e[0], e[1]) + tuple(e[2:]) for e in entries], chunk_bytes,
                                    lanes, tile, codebook, tile_order)
    if blob is None:
        blob = torch.empty(cap, dtype=torch.uint8, device=dev)
    if workspace is None:
        workspace = torch.empty(wsb, dtype=torch.uint8, device=dev)
    if size is None:
        size = torch.zeros(1, dtype=torch.int64, device=dev)
    if stream is None:
        stream = torch.cuda.current_stream(dev)
    arr = _dtensors(entries)
    prm = _params(chunk_bytes, lanes, tile, codebook, tile_order)
    rc = lib().wc_encode_device(arr, len(entries), C.byref(prm), C.c_void_p(blob.data_ptr()),
                                blob.numel(), C.c_void_p(workspace.data_ptr()), workspace.numel(),
                                C.c_void_p(stream.cuda_stream or None),
                                C.c_void_p(size.data_ptr()))
    if rc:
        raise WcError("wc_encode_device", rc)
    return blob, size


def gemm_torch(blob: Blob, dev_blob, tensors, xs, ys=None, workspace=None, stream=None, err=None):
    """wc_gemm into float32 tensors: ys[i] += xs[i] @ W_i^T (ys zeroed and
    returned if None; the workspace is allocated if None)."""
    import torch
    m = xs[0].shape[0]
    for x in xs:
        if x.dtype != torch.bfloat16 or not x.is_contiguous() or x.shape[0] != m:
            raise ValueError("xs must be contiguous bfloat16 tensors with equal row counts")
    if ys is None:
        ys = [torch.zeros((m, blob.shape(t)[0]), dtype=torch.float32, device=x.device)
              for t, x in zip(tensors, xs)]
    need = gemm_workspace_bytes(blob, list(tensors), [x.data_ptr() for x in xs], m)
    if workspace is None:
        workspace = torch.empty(max(need, 256), dtype=torch.uint8, device=xs[0].device)
    if stream is None:
        stream = torch.cuda.current_stream(xs[0].device)
    gemm(blob, dev_blob.data_ptr(), list(tensors), [x.data_ptr() for x in xs], m,
         [y.data_ptr() for y in ys], workspace.data_ptr(), workspace.numel(), stream.cuda_stream,
         err.data_ptr() if err is not None else 0)
    return ys


def gemm_i8_torch(blob: Blob, dev_blob, tensors, xs, ys=None, stream=None, err=None):
    """wc_gemm_i8 into int32 tensors: ys[i] += xs[i] @ W_i^T for int8 xs and
    int8 W_i = tensor tensors[i] (ys zeroed and returned if None)."""
    import torch
    m = xs[0].shape[0]
    for x in xs:
        if x.dtype != torch.int8 or not x.is_contiguous() or x.shape[0] != m:
            raise ValueError("xs must be contiguous int8 tensors with equal row counts")
    if ys is None:
        ys = [torch.zeros((m, blob.shape(t)[0]), dtype=torch.int32, device=x.device)
              for t, x in zip(tensors, xs)]
    if stream is None:
        stream = torch.cuda.current_stream(xs[0].device)
    gemm_i8(blob, dev_blob.data_ptr(), list(tensors), [x.data_ptr() for x in xs], m,
            [y.data_ptr() for y in ys], stream.cuda_stream, err.data_ptr() if err is not None else 0)
    return ys


def _codes_shape(blob: Blob, t: int):
    """(N, K) of a 4-bit weight tensor in codes: a nibble tensor's own shape, or
    twice the columns of a byte tensor holding the packed codes."""
    n, k = blob.shape(t)
    if blob.dtype(t) == "u8":
        k *= 2
    return n, k


def _check_jobs(blob: Blob, tensors, xs, m: int):
    """xs: one contiguous bf16 m x K tensor per job, K the weights' code count."""
    import torch
    if len(xs) != len(tensors):
        raise ValueError("one x per job")
    for t, x in zip(tensors, xs):
        if x.dtype != torch.bfloat16 or not x.is_contiguous() or x.dim() != 2 or x.shape[0] != m:
            raise ValueError("xs must be contiguous 2-D bfloat16 tensors with equal row counts")
        if not 0 <= t < blob.n_tensors:
            raise ValueError(f"tensor index {t} out of range")
        k = _codes_shape(blob, t)[1]
        if x.shape[1] != k:
            raise ValueError(f"tensor {t}: x has {x.shape[1]} columns, the weights {k}")


def gemv_mx_torch(blob: Blob, dev_blob, tensors, scales, xs, ys=None, stream=None, err=None):
    """wc_gemv_mx into float32 tensors: ys[i] += xs[i] @ W_i^T for MXFP4 W_i =
    tensor tensors[i] with e8m0 scales `scales[i]` (uint8 device tensors of
    N x K/32); ys zeroed and returned if None."""
    import torch
    m = xs[0].shape[0]
    _check_jobs(blob, tensors, xs, m)
    if len(scales) != len(tensors):
        raise ValueError("one scale tensor per job")
    for t, sc in zip(tensors, scales):
        n, k = _codes_shape(blob, t)
        if sc.dtype != torch.uint8 or not sc.is_contiguous():
            raise ValueError("scales must be contiguous uint8 tensors")
        if sc.numel() != n * (k // 32):
            raise ValueError(f"tensor {t}: {sc.numel()} scale bytes, the weights need N * K/32 = "
                             f"{n * (k // 32)}")
    if ys is None:
        ys = [torch.zeros((m, blob.shape(t)[0]), dtype=torch.float32, device=x.device)
              for t, x in zip(tensors, xs)]
    if stream is None:
        stream = torch.cuda.current_stream(xs[0].device)
    gemv_mx(blob, dev_blob.data_ptr(), list(tensors), [sc.data_ptr() for sc in scales],
            [x.data_ptr() for x in xs], m, [y.data_ptr() for y in ys], stream.cuda_stream,
            err.data_ptr() if err is not None else 0)
    return ys


def gemv_w4_torch(blob: Blob, dev_blob, tensors, scales, zeros, xs, ys=None, stream=None,
                  err=None):
    """wc_gemv_w4 into float32 tensors: ys[i] += xs[i] @ W_i^T for int4 W_i with fp16
    scales `scales[i]` (device tensors holding N x K/128 binary16 words, of any
    element type) and zero points `zeros[i]` (uint8 device tensors of one byte per
    group, or None for two's-complement codes; `zeros` None: all two's-complement);
    ys zeroed and returned if None.  Every tensor's size is checked against the
    weights' shape before the launch (ValueError), since the kernel sizes its reads
    from the blob, not from the tensors passed."""
    import torch
    m = xs[0].shape[0]
    _check_jobs(blob, tensors, xs, m)
    if len(scales) != len(tensors) or (zeros is not None and len(zeros) != len(tensors)):
        raise ValueError("one scale tensor (and one zero-point entry, if any) per job")
    for i, t in enumerate(tensors):
        n, k = _codes_shape(blob, t)
        sc = scales[i]
        if not sc.is_contiguous() or sc.data_ptr() % 2:
            raise ValueError("scales must be contiguous and 2-byte aligned")
        if sc.numel() * sc.element_size() != 2 * n * (k // 128):
            raise ValueError(f"tensor {t}: {sc.numel() * sc.element_size()} bytes of scales, the "
                             f"weights need N * K/128 = {n * (k // 128)} fp16 words")
        z = None if zeros is None else zeros[i]
        if z is not None:
            if z.dtype != torch.uint8 or not z.is_contiguous():
                raise ValueError("zero points must be contiguous uint8 tensors, one byte a group")
            if z.numel() != n * (k // 128):
                raise ValueError(f"tensor {t}: {z.numel()} zero points, the weights need one "
                                 f"byte per group, N * K/128 = {n * (k // 128)} (packed "
                                 "nibbles must be unpacked first)")
    if ys is None:
        ys = [torch.zeros((m, blob.shape(t)[0]), dtype=torch.float32, device=x.device)
              for t, x in zip(tensors, xs)]
    if stream is None:
        stream = torch.cuda.current_stream(xs[0].device)
    zp = None if zeros is None else [z.data_ptr() if z is not None else 0 for z in zeros]
    gemv_w4(blob, dev_blob.data_ptr(), list(tensors), [s.data_ptr() for s in scales], zp,
            [x.data_ptr() for x in xs], m, [y.data_ptr() for y in ys], stream.cuda_stream,
            err.data_ptr() if err is not None else 0)
    return ys
