"""CPU oracle of the chunked rANS weight codec -- TEST INFRASTRUCTURE ONLY.

Python view (ctypes) of ``wc_oracle.c``: a plain, single-threaded statement
of what the GPU decode path must reproduce.  Only ``tests/``, the package
smoke check and the benchmark's CPU-baseline leg may import this module.  It
never imports the HIP package and the HIP package never imports it.

Functions cite the paper passage they follow in ``wc_oracle.c``.
"""

from __future__ import annotations

import ctypes as C
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "wc_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

DTYPES = {"bf16": 1, "fp16": 2, "u8": 3, "u4": 4, "fp8_e4m3": 5, "fp8_e5m2": 6, "fp4_e2m1": 7}
_NIBBLE = ("u4", "fp4_e2m1")
_BYTE = ("u8", "fp8_e4m3", "fp8_e5m2")


def build(force: bool = False) -> str:
    """Compile the oracle with the host C compiler (plain C99, -O2)."""
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + f".tmp{os.getpid()}"
        subprocess.check_call(["gcc", "-O2", "-std=c99", "-Wall", "-fPIC", "-shared", _SRC,
                               "-o", tmp, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


_lib = None


class Stats(C.Structure):
    _fields_ = [("n_fields", C.c_uint32), ("alphabet", C.c_uint32 * 2),
                ("count", C.c_uint64 * 2), ("hist", (C.c_uint64 * 256) * 2),
                ("H", C.c_double * 2), ("H_joint16", C.c_double),
                ("bound_bytes", C.c_double), ("bound_bytes_raw8", C.c_double)]


class _Tensor(C.Structure):
    _fields_ = [("data", C.c_void_p), ("nbytes", C.c_uint64), ("dtype", C.c_uint32),
                ("rows", C.c_uint64), ("cols", C.c_uint64)]


def lib():
    global _lib
    if _lib is None:
        build()
        L = C.CDLL(_LIB)
        u8p = C.POINTER(C.c_uint8)
        L.orc_coded16.restype = C.c_uint8
        L.orc_coded16.argtypes = [C.c_uint16]
        L.orc_raw16.restype = C.c_uint8
        L.orc_raw16.argtypes = [C.c_uint16]
        L.orc_merge16.restype = C.c_uint16
        L.orc_merge16.argtypes = [C.c_uint8, C.c_uint8]
        L.orc_symbols.argtypes = [C.c_uint32, C.c_void_p, C.c_uint64, C.c_void_p, C.c_void_p]
        L.orc_histogram.argtypes = [C.c_void_p, C.c_uint64, C.c_void_p]
        L.orc_histogram.restype = None
        L.orc_entropy.restype = C.c_double
        L.orc_entropy.argtypes = [C.c_void_p, C.c_uint32]
        L.orc_analyze.argtypes = [C.c_uint32, C.c_void_p, C.c_uint64, C.POINTER(Stats)]
        L.orc_normalise.argtypes = [C.c_void_p, C.c_uint32, C.c_void_p]
        L.orc_encode_stream.argtypes = [C.c_void_p, C.c_uint64, C.c_void_p, C.c_uint32,
                                        C.c_uint32, C.c_uint32, C.c_void_p, C.c_uint32,
                                        C.c_void_p, C.c_void_p, C.c_uint64,
                                        C.POINTER(C.c_uint64), C.POINTER(C.c_uint32)]
        L.orc_decode_stream.argtypes = [C.c_void_p, C.c_uint32, C.c_void_p, C.c_uint64,
                                        C.c_uint64, C.c_void_p, C.c_uint32, C.c_uint32,
                                        C.c_uint32, C.c_uint32, C.c_void_p, C.c_void_p]
        L.orc_encode_blob.argtypes = [C.POINTER(_Tensor), C.c_uint32, C.c_uint32, C.c_uint32,
                                      C.c_uint32, C.c_uint32, C.c_uint32, C.c_uint32,
                                      C.POINTER(u8p), C.POINTER(C.c_uint64)]
        L.orc_gemv_bf16.argtypes = [C.c_void_p, C.c_uint64, C.c_uint64, C.c_void_p, C.c_uint32,
                                    C.c_void_p, C.c_void_p]
        L.orc_gemm_i8.argtypes = [C.c_void_p, C.c_uint64, C.c_uint64, C.c_void_p, C.c_uint32,
                                  C.c_void_p]
        L.orc_gemv_fp8.argtypes = [C.c_void_p, C.c_uint64, C.c_uint64, C.c_void_p, C.c_uint32,
                                   C.c_uint32, C.c_void_p, C.c_void_p]
        L.orc_e4m3_value.argtypes = [C.c_uint8]
        L.orc_e4m3_value.restype = C.c_double
        L.orc_e5m2_value.argtypes = [C.c_uint8]
        L.orc_e5m2_value.restype = C.c_double
        L.orc_e2m1_value.argtypes = [C.c_uint8]
        L.orc_e2m1_value.restype = C.c_double
        L.orc_e8m0_value.argtypes = [C.c_uint8]
        L.orc_e8m0_value.restype = C.c_double
        L.orc_fp16_value.argtypes = [C.c_uint16]
        L.orc_fp16_value.restype = C.c_double
        L.orc_gemv_int4.argtypes = [C.c_void_p, C.c_void_p, C.c_void_p, C.c_uint64, C.c_uint64,
                                    C.c_void_p, C.c_uint32, C.c_void_p, C.c_void_p]
        L.orc_gemv_mxfp4.argtypes = [C.c_void_p, C.c_void_p, C.c_uint64, C.c_uint64, C.c_void_p,
                                     C.c_uint32, C.c_void_p, C.c_void_p]
        L.orc_free.argtypes = [C.c_void_p]
        L.orc_free.restype = None
        L.orc_blob_tensors.argtypes = [C.c_void_p, C.c_uint64, C.POINTER(C.c_uint32)]
        L.orc_blob_tensor_info.argtypes = [C.c_void_p, C.c_uint64, C.c_uint32,
                                           C.POINTER(C.c_uint64), C.POINTER(C.c_uint32),
                                           C.POINTER(C.c_uint64), C.POINTER(C.c_uint32)]
        L.orc_decode_blob.argtypes = [C.c_void_p, C.c_uint64, C.POINTER(C.c_void_p)]
        L.orc_decode_chunks.argtypes = [C.c_void_p, C.c_uint64, C.c_uint32, C.c_uint64,
                                        C.c_uint64, C.c_void_p]
        L.orc_metadata_bytes.restype = C.c_double
        L.orc_metadata_bytes.argtypes = [C.c_uint64] * 4 + [C.c_uint32]
        _lib = L
    return _lib


class OracleError(RuntimeError):
    def __init__(self, rc, what):
        super().__init__(f"oracle {what} failed with status {rc}")
        self.rc = rc


def _ptr(a: np.ndarray):
    return a.ctypes.data_as(C.c_void_p)


def _bytes_view(data) -> np.ndarray:
    a = np.ascontiguousarray(data)
    return a.view(np.uint8).reshape(-1)


# --- field split ------------------------------------------------------------

def coded16(w: int) -> int:
    return lib().orc_coded16(w)


def raw16(w: int) -> int:
    return lib().orc_raw16(w)


def merge16(coded: int, raw: int) -> int:
    return lib().orc_merge16(coded, raw)


def symbols(dtype: str, data):
    """(coded symbols, raw bytes or None) of a tensor's storage bytes."""
    b = _bytes_view(data)
    dt = DTYPES[dtype]
    n = 2 * b.size if dtype in _NIBBLE else (b.size if dtype in _BYTE else b.size // 2)
    coded = np.empty(max(n, 1), np.uint8)
    raw = np.empty(max(n, 1), np.uint8)
    rc = lib().orc_symbols(dt, _ptr(b), b.size, _ptr(coded), _ptr(raw))
    if rc:
        raise OracleError(rc, "symbols")
    return coded[:n], (raw[:n] if dtype in ("bf16", "fp16") else None)


# --- statistics --------------------------------------------------------------

def histogram(sym: np.ndarray) -> np.ndarray:
    s = np.ascontiguousarray(sym, dtype=np.uint8)
    h = np.zeros(256, np.uint64)
    lib().orc_histogram(_ptr(s), s.size, _ptr(h))
    return h


def entropy(hist, alphabet: int | None = None) -> float:
    h = np.ascontiguousarray(hist, dtype=np.uint64)
    return lib().orc_entropy(_ptr(h), alphabet or h.size)


def analyze(dtype: str, data) -> dict:
    b = _bytes_view(data)
    st = Stats()
    rc = lib().orc_analyze(DTYPES[dtype], _ptr(b), b.size, C.byref(st))
    if rc:
        raise OracleError(rc, "analyze")
    nf = st.n_fields
    return {
        "n_fields": nf,
        "alphabet": [st.alphabet[i] for i in range(nf)],
        "count": [st.count[i] for i in range(nf)],
        "hist": [np.array(st.hist[i][:st.alphabet[i]], np.uint64) for i in range(nf)],
        "H": [st.H[i] for i in range(nf)],
        "H_joint16": st.H_joint16,
        "bound_bytes": st.bound_bytes,
        "bound_bytes_raw8": st.bound_bytes_raw8,
    }


def normalise(hist, alphabet: int | None = None) -> np.ndarray:
    h = np.ascontiguousarray(hist, dtype=np.uint64)
    a = alphabet or h.size
    f = np.zeros(256, np.uint32)
    rc = lib().orc_normalise(_ptr(h), a, _ptr(f))
    if rc:
        raise OracleError(rc, "normalise")
    return f[:a]


# --- one interleaved rANS stream --------------------------------------------

def encode_stream(sym, freq, lanes: int, group: int, init=None, skip: int = 0):
    """(states, words) of one chunk coded with `lanes` lanes of `group` symbols.

    `init`: each lane's start state (default 2^16); steps below `skip` of
    every lane are left out of the coding."""
    s = np.ascontiguousarray(sym, dtype=np.uint8)
    f = np.ascontiguousarray(freq, dtype=np.uint32)
    cap = s.size + 1
    words = np.empty(cap, np.uint16)
    states = np.empty(max(lanes, 1), np.uint32)
    ini = None if init is None else np.ascontiguousarray(init, dtype=np.uint32)
    nw = C.c_uint64()
    na = C.c_uint32()
    rc = lib().orc_encode_stream(_ptr(s), s.size, _ptr(f), f.size, lanes, group,
                                 None if ini is None else _ptr(ini), skip, _ptr(states),
                                 _ptr(words), cap, C.byref(nw), C.byref(na))
    if rc:
        raise OracleError(rc, "encode_stream")
    return states[:na.value].copy(), words[:nw.value].copy()


def decode_stream(states, words, n: int, freq, lanes: int, group: int, skip: int = 0,
                  want_final: bool = False):
    """Decoded symbols (steps below `skip` left at 0), or raises OracleError(-3)
    if the checks fail.  Every lane must end at 2^16, unless want_final: then
    the end states are returned too, (symbols, states), for the caller to check."""
    st = np.ascontiguousarray(states, dtype=np.uint32)
    w = np.ascontiguousarray(words, dtype=np.uint16)
    f = np.ascontiguousarray(freq, dtype=np.uint32)
    out = np.zeros(max(n, 1), np.uint8)
    fin = np.zeros(max(st.size, 1), np.uint32)
    rc = lib().orc_decode_stream(_ptr(st), st.size, _ptr(w), w.size, n, _ptr(f), f.size, lanes,
                                 group, skip, _ptr(fin) if want_final else None, _ptr(out))
    if rc:
        raise OracleError(rc, "decode_stream")
    return (out[:n], fin[:st.size].copy()) if want_final else out[:n]


# --- blobs -------------------------------------------------------------------

def encode(tensors, chunk_bytes: int = 65536, lanes: int = 64, tile=(0, 0),
           codebook: str = "tensor", tile_order: int = 0) -> bytes:
    """Blob bytes of a list of (dtype, storage array[, (rows, cols)]) entries.

    `tile` = (rows, cols) cuts every tensor whose shape (in symbol elements:
    16-bit words, bytes or nibbles) the tile divides into one chunk per tile;
    the others use `chunk_bytes`.  tile_order 0 keeps each tile row-major, 1
    lists its lane-groups k-block by k-block (column blocks).  codebook
    "layer" shares one table among all tensors of a dtype.
    """
    keep = []
    arr = (_Tensor * len(tensors))()
    for i, entry in enumerate(tensors):
        dt, data = entry[0], entry[1]
        rows, cols = entry[2] if len(entry) > 2 and entry[2] is not None else (0, 0)
        b = _bytes_view(data)
        keep.append(b)
        arr[i].data = b.ctypes.data if b.size else None
        arr[i].nbytes = b.size
        arr[i].dtype = DTYPES[dt]
        arr[i].rows, arr[i].cols = rows, cols
    out = C.POINTER(C.c_uint8)()
    size = C.c_uint64()
    shared = {"tensor": 0, "layer": 1}[codebook]
    rc = lib().orc_encode_blob(arr, len(tensors), chunk_bytes, lanes, tile[0], tile[1],
                               tile_order, shared, C.byref(out), C.byref(size))
    if rc:
        raise OracleError(rc, "encode")
    try:
        return C.string_at(out, size.value)
    finally:
        lib().orc_free(out)


def _blob_array(blob) -> np.ndarray:
    return np.frombuffer(blob, dtype=np.uint8) if not isinstance(blob, np.ndarray) else blob


def tensor_info(blob):
    b = _blob_array(blob)
    n = C.c_uint32()
    rc = lib().orc_blob_tensors(_ptr(b), b.size, C.byref(n))
    if rc:
        raise OracleError(rc, "blob header")
    info = []
    for t in range(n.value):
        ob, dt, nc = C.c_uint64(), C.c_uint32(), C.c_uint64()
        tile = (C.c_uint32 * 4)()
        rc = lib().orc_blob_tensor_info(_ptr(b), b.size, t, C.byref(ob), C.byref(dt),
                                        C.byref(nc), tile)
        if rc:
            raise OracleError(rc, "tensor info")
        info.append({"out_bytes": ob.value, "dtype": dt.value, "n_chunks": nc.value,
                     "tile": (tile[0], tile[1]), "chunk_bytes": tile[2],
                     "tile_order": tile[3]})
    return info


def decode(blob):
    """List of decoded tensors (uint8 storage bytes)."""
    b = _blob_array(blob)
    info = tensor_info(b)
    outs = [np.zeros(max(i["out_bytes"], 1), np.uint8) for i in info]
    ptrs = (C.c_void_p * len(outs))(*[o.ctypes.data for o in outs])
    rc = lib().orc_decode_blob(_ptr(b), b.size, ptrs)
    if rc:
        raise OracleError(rc, "decode")
    return [o[:i["out_bytes"]] for o, i in zip(outs, info)]


def decode_chunks(blob, tensor: int, c0: int, c1: int, out: np.ndarray | None = None):
    """Decode chunks [c0, c1) of one tensor into `out` (whole-tensor buffer)."""
    b = _blob_array(blob)
    info = tensor_info(b)[tensor]
    if out is None:
        out = np.zeros(max(info["out_bytes"], 1), np.uint8)
    rc = lib().orc_decode_chunks(_ptr(b), b.size, tensor, c0, c1, _ptr(out))
    if rc:
        raise OracleError(rc, "decode_chunks")
    return out


def metadata_bytes(rows: int, cols: int, tile_r: int, tile_c: int, b: int = 12) -> float:
    return lib().orc_metadata_bytes(rows, cols, tile_r, tile_c, b)



def gemv_bf16(w, x):
    """(y, sum |x w|) in fp64: y[m, n] = sum_k x[m, k] * w[n, k] for bf16 storage
    words w (rows x cols) and x (M x cols), summed in k order."""
    w = np.ascontiguousarray(w, dtype=np.uint16)
    x = np.ascontiguousarray(x, dtype=np.uint16)
    rows, cols = w.shape
    M = x.shape[0]
    assert x.shape[1] == cols
    y = np.empty((M, rows), np.float64)
    a = np.empty((M, rows), np.float64)
    rc = lib().orc_gemv_bf16(_ptr(w), rows, cols, _ptr(x), M, _ptr(y), _ptr(a))
    if rc:
        raise OracleError(rc, "gemv")
    return y, a


def gemm_i8(w, x):
    """y[m, n] = sum_k x[m, k] * w[n, k] exactly (int64) for int8 w (rows x
    cols) and int8 x (M x cols)."""
    w = np.ascontiguousarray(w, dtype=np.int8)
    x = np.ascontiguousarray(x, dtype=np.int8)
    rows, cols = w.shape
    M = x.shape[0]
    assert x.shape[1] == cols
    y = np.empty((M, rows), np.int64)
    rc = lib().orc_gemm_i8(_ptr(w), rows, cols, _ptr(x), M, _ptr(y))
    if rc:
        raise OracleError(rc, "gemm_i8")
    return y


def e4m3_value(v: int) -> float:
    """The value of one OCP e4m3 byte (NaN for the two NaN patterns)."""
    return lib().orc_e4m3_value(v)


def e5m2_value(v: int) -> float:
    """The value of one OCP e5m2 byte (+-inf, NaN for the exponent-31 patterns)."""
    return lib().orc_e5m2_value(v)


def e2m1_value(nibble: int) -> float:
    """The value of one fp4 e2m1 code (low 4 bits)."""
    return lib().orc_e2m1_value(nibble)


def e8m0_value(e: int) -> float:
    """The value of one e8m0 scale byte: 2^(e - 127), NaN for 255."""
    return lib().orc_e8m0_value(e)


def gemv_mxfp4(w, scales, x):
    """(y, sum |x w|) in fp64 for MXFP4 weights: w the packed e2m1 codes
    (rows x cols/2 bytes, even element in the low nibble), scales the e8m0
    bytes (rows x cols/32), x bf16 storage words (M x cols)."""
    w = np.ascontiguousarray(w, dtype=np.uint8)
    scales = np.ascontiguousarray(scales, dtype=np.uint8)
    x = np.ascontiguousarray(x, dtype=np.uint16)
    rows, cols = w.shape[0], 2 * w.shape[1]
    M = x.shape[0]
    assert x.shape[1] == cols and scales.shape == (rows, cols // 32)
    y = np.empty((M, rows), np.float64)
    a = np.empty((M, rows), np.float64)
    rc = lib().orc_gemv_mxfp4(_ptr(w), _ptr(scales), rows, cols, _ptr(x), M, _ptr(y), _ptr(a))
    if rc:
        raise OracleError(rc, "gemv_mxfp4")
    return y, a


def fp16_value(h: int) -> float:
    """The value of one IEEE binary16 storage word."""
    return lib().orc_fp16_value(h)


def gemv_int4(w, scales, zeros, x):
    """(y, sum |x w|) in fp64 for group-quantised int4 weights: w the packed
    codes (rows x cols/2 bytes, even element low), scales fp16 storage words
    (rows x cols/128), zeros one byte per group (rows x cols/128; codes
    unsigned, weight s (q - z)) or None (two's-complement codes, weight s q),
    x bf16 storage words (M x cols)."""
    w = np.ascontiguousarray(w, dtype=np.uint8)
    scales = np.ascontiguousarray(scales, dtype=np.uint16)
    x = np.ascontiguousarray(x, dtype=np.uint16)
    rows, cols = w.shape[0], 2 * w.shape[1]
    M = x.shape[0]
    assert x.shape[1] == cols and scales.shape == (rows, cols // 128)
    zp = None
    if zeros is not None:
        zeros = np.ascontiguousarray(zeros, dtype=np.uint8)
        assert zeros.shape == (rows, cols // 128)
        zp = _ptr(zeros)
    y = np.empty((M, rows), np.float64)
    a = np.empty((M, rows), np.float64)
    rc = lib().orc_gemv_int4(_ptr(w), _ptr(scales), zp, rows, cols, _ptr(x), M, _ptr(y), _ptr(a))
    if rc:
        raise OracleError(rc, "gemv_int4")
    return y, a


FP8_FORMATS = {"e4m3": 0, "e5m2": 1}


def gemv_fp8(w, x, fmt: str = "e4m3"):
    """(y, sum |x w|) in fp64: y[m, n] = sum_k x[m, k] * fp8(w[n, k]) for fp8
    bytes w (rows x cols) of format `fmt` ("e4m3" or "e5m2") and bf16 storage
    words x (M x cols)."""
    w = np.ascontiguousarray(w, dtype=np.uint8)
    x = np.ascontiguousarray(x, dtype=np.uint16)
    rows, cols = w.shape
    M = x.shape[0]
    assert x.shape[1] == cols
    y = np.empty((M, rows), np.float64)
    a = np.empty((M, rows), np.float64)
    rc = lib().orc_gemv_fp8(_ptr(w), rows, cols, _ptr(x), M, FP8_FORMATS[fmt], _ptr(y), _ptr(a))
    if rc:
        raise OracleError(rc, "gemv_fp8")
    return y, a
