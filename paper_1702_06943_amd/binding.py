"""ctypes binding of libtoc.so: argument marshalling only.

Every function has the name of the C entry point it calls (include/toc.h) and
raises TocError on any status other than TOC_OK.  Host arrays are numpy arrays;
device arrays are torch tensors on the GPU, used only for their pointers; the
stream defaults to torch's current stream.  Nothing here computes any part of the
compression or of the products.
"""

from __future__ import annotations

import ctypes as C
import os

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libtoc.so")
# A host-sanitizer build of the same library (tests only, see sanitize.py) is
# loaded instead when TOC_LIB_PATH names it.
LIB_PATH = os.environ.get("TOC_LIB_PATH", LIB_PATH)

TOC_OK, TOC_EINVAL, TOC_ENOMEM, TOC_ESIZE, TOC_EDEVICE, TOC_EUNSUPPORTED = range(6)
TOC_UPLOAD_KEEP_DEAD = 1
TOC_UPLOAD_HOST = 2
TOC_OP_RIGHT, TOC_OP_LEFT, TOC_OP_DECODE = 0, 1, 2
TOC_MAP_SCALE, TOC_MAP_SQUARE = 0, 1
TOC_MGD_LINEAR, TOC_MGD_LOGISTIC, TOC_MGD_HINGE = 0, 1, 2
TOC_ENCDEV_ROWPTR, TOC_ENCDEV_SIZE, TOC_ENCDEV_COLUMN, TOC_ENCDEV_VALUE = range(1, 5)
(TOC_CPRIME_LAYOUT, TOC_CPRIME_VALUE_INDEX, TOC_CPRIME_STARTS, TOC_CPRIME_CODE,
 TOC_CPRIME_NODES, TOC_CPRIME_ROWS, TOC_LEVEL_D, TOC_LEVEL_DEPTH, TOC_LEVEL_LIVE) = range(1, 10)
TOC_CPRIME_COLUMN = 10
TOC_INGEST_CHANGED = 11
TOC_NOALLOC_SCRATCH_BYTES = 64 << 20
STATUS_NAMES = {0: "TOC_OK", 1: "TOC_EINVAL", 2: "TOC_ENOMEM", 3: "TOC_ESIZE",
                4: "TOC_EDEVICE", 5: "TOC_EUNSUPPORTED"}


class TocError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {msg}")
        self.status = status


class EncInfo(C.Structure):
    _fields_ = [("n_rows", C.c_int32), ("n_cols", C.c_int32), ("nnz", C.c_int64),
                ("n_first", C.c_int64), ("n_codes", C.c_int64), ("n_nodes", C.c_int64),
                ("n_live", C.c_int64), ("n_deep", C.c_int64), ("max_depth", C.c_int32),
                ("reserved", C.c_int32), ("phys_bytes", C.c_int64),
                ("canon_bytes", C.c_int64)]


class DevInfo(C.Structure):
    _fields_ = [("n_batches", C.c_int64), ("n_rows", C.c_int64), ("n_cols", C.c_int32),
                ("max_depth", C.c_int32), ("nnz", C.c_int64), ("n_codes", C.c_int64),
                ("n_stored", C.c_int64), ("n_deep", C.c_int64), ("canon_bytes", C.c_int64),
                ("image_bytes", C.c_int64)]


class PhysInfo(C.Structure):
    _fields_ = [(n, C.c_int64) for n in
                ("n_rows", "n_first", "n_codes", "n_unique", "n_nodes", "max_col")]


class Layout(C.Structure):
    _fields_ = [(n, C.c_int64) for n in
                ("batches", "level", "key", "link", "span", "dcodes", "occ_off", "tlist",
                 "dtiles", "cols", "tchild", "centry", "cval", "end")]


# records of the image's key and link arrays (toc_key, toc_link)
KEY_DTYPE = np.dtype([("col", "<u4"), ("val", "<f4")])
LINK_DTYPE = np.dtype([("parent", "<u4"), ("depth", "<u4")])


BATCH_DTYPE = np.dtype([
    ("code_base", "<i8"), ("d_base", "<i8"), ("row_base", "<i8"), ("span_base", "<i8"),
    ("nnz_base", "<i8"), ("deep_base", "<i8"), ("tree_base", "<i8"), ("lvl_base", "<i8"),
    ("n_rows", "<i4"), ("n_codes", "<i4"), ("n_lvl1", "<i4"), ("n_int1", "<i4"),
    ("n_levels", "<i4"), ("n_d", "<i4"), ("n_ucols", "<i4"), ("pad", "<i4")])

_lib = None


def lib():
    """The loaded libtoc.so; raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                           "`python -m paper_1702_06943_amd.build`")
    # torch ships its own HIP runtime under the same soname; loading torch first
    # makes libtoc bind to that one, so that streams and device pointers agree.
    try:
        import torch  # noqa: F401
    except ImportError:
        pass
    L = C.CDLL(LIB_PATH)
    P, I32, I64, U32, SZ = C.c_void_p, C.c_int32, C.c_int64, C.c_uint32, C.c_size_t
    sig = {
        "toc_encode": [I32, I32, P, P, P, P],
        "toc_encode_batches": [I64, P, I32, P, P, P, I32, P],
        "toc_enc_info_get": [P, P],
        "toc_enc_export": [P, P, P, P, P],
        "toc_upload_size": [P, I64, U32, P],
        "toc_upload": [P, I64, U32, P, SZ, P, P],
        "toc_dev_info_get": [P, P],
        "toc_dev_layout_get": [P, P],
        "toc_workspace_size": [P, I32, I32, P, P],
        "toc_right_mul": [P, P, I32, I64, P, I64, P, SZ, P],
        "toc_left_mul": [P, P, I32, I64, P, I64, I32, P, SZ, P],
        "toc_left_mul_noalloc": [P, P, I32, I64, P, I64, I32, P],
        "toc_decode_csr": [P, P, P, P, P],
        "toc_map_values": [P, I32, C.c_float, P],
        "toc_decode_dense": [P, C.c_float, P, I64, P],
        "toc_enc_pack_size": [P, P],
        "toc_enc_pack": [P, P, SZ],
        "toc_phys_info_get": [P, SZ, P],
        "toc_cprime_workspace_size": [I64, I64, P],
        "toc_cprime_build": [P, P, P, I64, I32, I32, P, P, P, P, P, P, SZ, P],
        "toc_mgd_epoch": [P, I64, I64, I32, C.c_float, P, P, P],
        "toc_mgd_workspace_size": [P, P],
        "toc_mgd_epoch_split": [P, I64, I64, I32, C.c_float, P, P, P, SZ, P],
        "toc_encode_device_workspace_size": [I64, I64, P],
        "toc_mlp_workspace_size": [P, I32, I32, I32, P],
        "toc_level_workspace_size": [I64, I64, P],
        "toc_level_right_mul": [P, P, P, P, P, I64, I32, I32, I64, P, P, P, P, P, P, P, P, P, P,
                                P, SZ, P],
        "toc_level_build": [P, P, P, P, I64, I32, P, P, P, P, P, P, P, P, P, P, P, P, P, P, SZ, P],
        "toc_mlp_epoch": [P, I64, I64, I32, I32, I32, P, P, P, P, P, P, P, C.c_float, P, SZ, P],
        "toc_encode_device": [I64, P, I32, P, P, P, I64, I64, P, P, P, P, P, P, P, SZ, P],
        "toc_ingest_workspace_size": [P, I64, I32, P, P],
        "toc_ingest_plan": [P, P, P, I64, I32, P, SZ, P, P, P],
        "toc_ingest_build": [P, P, P, P, SZ, P, SZ, P],
    }
    for name, args in sig.items():
        f = getattr(L, name)
        f.argtypes = args
        f.restype = C.c_int
    L.toc_enc_free.argtypes = [P]
    L.toc_enc_free.restype = None
    L.toc_dev_free.argtypes = [P]
    L.toc_dev_free.restype = None
    L.toc_last_error.argtypes = []
    L.toc_last_error.restype = C.c_char_p
    _lib = L
    return L


def _check(status):
    if status != TOC_OK:
        raise TocError(status, lib().toc_last_error().decode(errors="replace"))


def _ptr(a):
    """Pointer of a numpy array or torch tensor (None -> NULL)."""
    if a is None:
        return None
    if isinstance(a, np.ndarray):
        return a.ctypes.data if a.size else None
    return a.data_ptr() if a.numel() else None


def _stream(stream):
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    if isinstance(stream, int):
        return stream
    return stream.cuda_stream


class Enc:
    """Owner of a toc_enc handle."""

    def __init__(self, handle):
        self.handle = handle

    def __del__(self):
        if getattr(self, "handle", None) and _lib is not None:
            _lib.toc_enc_free(self.handle)
            self.handle = None


class Dev:
    """Owner of a toc_dev descriptor; keeps the image buffer alive."""

    def __init__(self, handle, buf):
        self.handle = handle
        self.buf = buf

    def __del__(self):
        if getattr(self, "handle", None) and _lib is not None:
            _lib.toc_dev_free(self.handle)
            self.handle = None


def _arr(x, dtype):
    return np.ascontiguousarray(np.asarray(x), dtype=dtype)


def toc_encode(n_rows, n_cols, rowptr, col, val):
    rowptr, col, val = _arr(rowptr, np.int64), _arr(col, np.int32), _arr(val, np.float32)
    h = C.c_void_p()
    _check(lib().toc_encode(int(n_rows), int(n_cols), _ptr(rowptr), _ptr(col), _ptr(val),
                            C.byref(h)))
    return Enc(h.value)


def toc_encode_batches(n_rows, n_cols, rowptr, col, val, n_threads=0):
    """n_rows: rows per batch; rowptr/col/val: one concatenated CSR."""
    n_rows = _arr(n_rows, np.int32)
    rowptr, col, val = _arr(rowptr, np.int64), _arr(col, np.int32), _arr(val, np.float32)
    nb = len(n_rows)
    handles = (C.c_void_p * max(nb, 1))()
    _check(lib().toc_encode_batches(nb, _ptr(n_rows), int(n_cols), _ptr(rowptr), _ptr(col),
                                    _ptr(val), int(n_threads), handles))
    return [Enc(handles[b]) for b in range(nb)]


def toc_enc_info_get(enc):
    info = EncInfo()
    _check(lib().toc_enc_info_get(enc.handle, C.byref(info)))
    return {f: getattr(info, f) for f, _ in EncInfo._fields_ if f != "reserved"}


def toc_enc_export(enc):
    """-> (I_col int32, I_val float32, D_rowptr int64, D_codes uint32), paper numbering."""
    info = toc_enc_info_get(enc)
    I_col = np.empty(info["n_first"], np.int32)
    I_val = np.empty(info["n_first"], np.float32)
    D_rowptr = np.empty(info["n_rows"] + 1, np.int64)
    D_codes = np.empty(info["n_codes"], np.uint32)
    _check(lib().toc_enc_export(enc.handle, _ptr(I_col), _ptr(I_val), D_rowptr.ctypes.data,
                                _ptr(D_codes)))
    return I_col, I_val, D_rowptr, D_codes


def _handles(encs):
    arr = (C.c_void_p * max(len(encs), 1))()
    for i, e in enumerate(encs):
        arr[i] = e.handle
    return arr


def toc_upload_size(encs, flags=0):
    n = C.c_size_t()
    _check(lib().toc_upload_size(_handles(encs), len(encs), flags, C.byref(n)))
    return n.value


def toc_upload(encs, buf, flags=0, stream=None):
    """buf: torch uint8 tensor on the GPU (or a numpy uint8 array with TOC_UPLOAD_HOST)."""
    if isinstance(buf, np.ndarray):
        nbytes, s = buf.nbytes, None
    else:
        nbytes, s = buf.numel() * buf.element_size(), _stream(stream)
    h = C.c_void_p()
    _check(lib().toc_upload(_handles(encs), len(encs), flags, _ptr(buf), nbytes, s,
                            C.byref(h)))
    return Dev(h.value, buf)


def toc_dev_info_get(dev):
    info = DevInfo()
    _check(lib().toc_dev_info_get(dev.handle, C.byref(info)))
    return {f: getattr(info, f) for f, _ in DevInfo._fields_}


def toc_dev_layout_get(dev):
    L = Layout()
    _check(lib().toc_dev_layout_get(dev.handle, C.byref(L)))
    return {f: getattr(L, f) for f, _ in Layout._fields_}


def toc_workspace_size(dev, op, k):
    n, mn = C.c_size_t(), C.c_size_t()
    _check(lib().toc_workspace_size(dev.handle, op, int(k), C.byref(n), C.byref(mn)))
    return n.value, mn.value


def _mat(t, name):
    """(pointer, leading dimension, k) of a row-major 2-D float32 device tensor."""
    import torch
    if t.dtype != torch.float32 or t.dim() != 2 or t.stride(1) != 1 or not t.is_cuda:
        raise TocError(TOC_EINVAL, f"{name} must be a 2-D float32 CUDA tensor with unit "
                                   "column stride")
    return t.data_ptr(), max(t.stride(0), t.shape[1]), t.shape[1]


def _nbytes(t):
    return 0 if t is None else t.numel() * t.element_size()


def toc_right_mul(dev, W, R, ws=None, stream=None):
    info = toc_dev_info_get(dev)
    wp, ldw, k = _mat(W, "W")
    rp, ldr, kr = _mat(R, "R")
    if W.shape[0] != info["n_cols"] or R.shape[0] != info["n_rows"] or kr != k:
        raise TocError(TOC_EINVAL, "W must be n_cols x k and R n_rows x k")
    _check(lib().toc_right_mul(dev.handle, wp, k, ldw, rp, ldr, _ptr(ws), _nbytes(ws),
                               _stream(stream)))


def toc_left_mul(dev, G, out, accumulate=False, ws=None, stream=None):
    """out: (n_batches * n_cols) x k, block b holding (G_b^T A_b)^T."""
    info = toc_dev_info_get(dev)
    gp, ldg, k = _mat(G, "G")
    op_, ldo, ko = _mat(out, "out")
    if (G.shape[0] != info["n_rows"] or out.shape[0] != info["n_batches"] * info["n_cols"]
            or ko != k):
        raise TocError(TOC_EINVAL, "G must be n_rows x k, out (n_batches*n_cols) x k")
    _check(lib().toc_left_mul(dev.handle, gp, k, ldg, op_, ldo, int(bool(accumulate)),
                              _ptr(ws), _nbytes(ws), _stream(stream)))


def toc_left_mul_noalloc(dev, G, out, accumulate=False, stream=None):
    """toc_left_mul with its workspace in the library's static device buffer
    (TOC_NOALLOC_SCRATCH_BYTES per GPU): no workspace argument, no allocation."""
    info = toc_dev_info_get(dev)
    gp, ldg, k = _mat(G, "G")
    op_, ldo, ko = _mat(out, "out")
    if (G.shape[0] != info["n_rows"] or out.shape[0] != info["n_batches"] * info["n_cols"]
            or ko != k):
        raise TocError(TOC_EINVAL, "G must be n_rows x k, out (n_batches*n_cols) x k")
    _check(lib().toc_left_mul_noalloc(dev.handle, gp, k, ldg, op_, ldo, int(bool(accumulate)),
                                      _stream(stream)))


def toc_decode_csr(dev, rowptr, col, val, stream=None):
    info = toc_dev_info_get(dev)
    if (rowptr.numel() != info["n_rows"] + 1 or col.numel() != info["nnz"]
            or val.numel() != info["nnz"]):
        raise TocError(TOC_EINVAL, "rowptr/col/val sizes do not match the image")
    _check(lib().toc_decode_csr(dev.handle, rowptr.data_ptr(), _ptr(col), _ptr(val),
                                _stream(stream)))


def toc_map_values(dev, op, c=1.0, stream=None):
    """In place: every key value v of the image becomes v*c (TOC_MAP_SCALE) or v*v."""
    _check(lib().toc_map_values(dev.handle, int(op), float(c), _stream(stream)))


def toc_decode_dense(dev, A, c=0.0, stream=None):
    """A: n_rows x lda float32 (lda >= n_cols) receives the dense batches plus c."""
    info = toc_dev_info_get(dev)
    ap, lda, ncols = _mat(A, "A")
    if A.shape[0] != info["n_rows"] or ncols < info["n_cols"]:
        raise TocError(TOC_EINVAL, "A must be n_rows x (>= n_cols)")
    _check(lib().toc_decode_dense(dev.handle, float(c), ap, lda, _stream(stream)))


def toc_enc_pack(enc):
    """The physical encoding (section 3.2) of one encoded batch, as uint8 bytes."""
    n = C.c_size_t()
    _check(lib().toc_enc_pack_size(enc.handle, C.byref(n)))
    out = np.empty(max(n.value, 1), np.uint8)
    _check(lib().toc_enc_pack(enc.handle, _ptr(out), n.value))
    return out[:n.value]


def toc_phys_info_get(blob):
    """Counts of one physical-encoding blob (numpy uint8, host)."""
    blob = _arr(blob, np.uint8)
    info = PhysInfo()
    _check(lib().toc_phys_info_get(_ptr(blob), blob.size, C.byref(info)))
    return {f: getattr(info, f) for f, _ in PhysInfo._fields_}


def toc_cprime_workspace_size(n_batches, n_nodes):
    n = C.c_size_t()
    _check(lib().toc_cprime_workspace_size(int(n_batches), int(n_nodes), C.byref(n)))
    return n.value


def toc_cprime_build(blobs, blob_off, node_off, max_rows, n_cols, parent, col, val, depth,
                     status, ws, stream=None):
    """blobs: device uint8 tensor of the concatenated blobs; blob_off, node_off: host
    int64 arrays of n_batches + 1 offsets; n_cols: columns of the encoded matrix (a
    column of I at or above it is TOC_CPRIME_COLUMN); parent, col, depth: device int32/uint32
    tensors and val a float32 tensor of node_off[-1] entries; status: device int32
    tensor of n_batches entries; ws: device tensor of toc_cprime_workspace_size
    bytes."""
    blob_off, node_off = _arr(blob_off, np.int64), _arr(node_off, np.int64)
    nb = blob_off.size - 1
    if node_off.size != nb + 1:
        raise TocError(TOC_EINVAL, "blob_off and node_off differ in length")
    n = int(node_off[-1]) if nb >= 0 else 0
    for t, name in ((parent, "parent"), (col, "col"), (val, "val"), (depth, "depth")):
        if t.numel() < n or t.element_size() != 4:
            raise TocError(TOC_EINVAL, f"{name} must hold {n} 4-byte entries")
    if status.numel() < nb or status.element_size() != 4:
        raise TocError(TOC_EINVAL, "status must hold one int32 per batch")
    if blobs.numel() < int(blob_off[-1]):
        raise TocError(TOC_EINVAL, "blobs shorter than blob_off[-1]")
    _check(lib().toc_cprime_build(_ptr(blobs), _ptr(blob_off), _ptr(node_off), nb, int(max_rows),
                                  int(n_cols), _ptr(parent), _ptr(col), _ptr(val), _ptr(depth), _ptr(status),
                                  _ptr(ws), ws.numel() * ws.element_size() if ws is not None else 0,
                                  _stream(stream)))


def _phys_infos(infos):
    arr = (PhysInfo * max(len(infos), 1))()
    for i, f in enumerate(infos):
        for name, _ in PhysInfo._fields_:
            setattr(arr[i], name, int(f[name]))
    return arr


def toc_ingest_workspace_size(infos, n_cols):
    """infos: toc_phys_info_get of each blob.  Returns (bytes for one range of all
    batches, least bytes that take the largest batch)."""
    n, mn = C.c_size_t(), C.c_size_t()
    _check(lib().toc_ingest_workspace_size(_phys_infos(infos), len(infos), int(n_cols),
                                           C.byref(n), C.byref(mn)))
    return n.value, mn.value


def toc_ingest_plan(blobs, blob_off, infos, n_cols, ws, stream=None):
    """blobs: device uint8 tensor of the concatenated blobs; blob_off: host int64
    array of len(infos) + 1 offsets; ws: device workspace tensor.  Returns
    (image bytes, planned Dev); build it with toc_ingest_build."""
    blob_off = _arr(blob_off, np.int64)
    if blob_off.size != len(infos) + 1:
        raise TocError(TOC_EINVAL, "blob_off must have one entry per blob plus one")
    if blobs.numel() < int(blob_off[-1]):
        raise TocError(TOC_EINVAL, "blobs shorter than blob_off[-1]")
    n, h = C.c_size_t(), C.c_void_p()
    _check(lib().toc_ingest_plan(_ptr(blobs), _ptr(blob_off), _phys_infos(infos), len(infos),
                                 int(n_cols), _ptr(ws), _nbytes(ws) if ws is not None else 0,
                                 _stream(stream), C.byref(n), C.byref(h)))
    return n.value, Dev(h.value, None)


def toc_ingest_build(dev, blobs, blob_off, buf, ws, stream=None):
    """Builds the planned image into buf (device uint8 tensor of at least the
    plan's bytes); dev then keeps buf alive."""
    blob_off = _arr(blob_off, np.int64)
    _check(lib().toc_ingest_build(dev.handle, _ptr(blobs), _ptr(blob_off), _ptr(buf), _nbytes(buf),
                                  _ptr(ws), _nbytes(ws) if ws is not None else 0, _stream(stream)))
    dev.buf = buf


def toc_mgd_epoch(dev, y, h, loss, lr, b0=0, n_batches=None, stream=None):
    """MGD steps over batches b0 .. b0+n_batches-1 (default: all from b0).  y: device
    float32 tensor of one label per row of the image; h: device float32 tensor of
    n_cols entries, updated in place."""
    info = toc_dev_info_get(dev)
    if n_batches is None:
        n_batches = info["n_batches"] - b0
    if y.numel() < info["n_rows"] or y.element_size() != 4:
        raise TocError(TOC_EINVAL, "y must hold one float32 per row")
    if h.numel() != info["n_cols"] or h.element_size() != 4:
        raise TocError(TOC_EINVAL, "h must hold n_cols float32")
    _check(lib().toc_mgd_epoch(dev.handle, int(b0), int(n_batches), int(loss), float(lr),
                               _ptr(y), _ptr(h), _stream(stream)))


def toc_mgd_workspace_size(dev):
    """Device workspace bytes toc_mgd_epoch_split needs for this image."""
    n = C.c_size_t()
    _check(lib().toc_mgd_workspace_size(dev.handle, C.byref(n)))
    return n.value


def toc_mgd_epoch_split(dev, y, h, loss, lr, ws, b0=0, n_batches=None, stream=None):
    """toc_mgd_epoch's steps, each split over many workgroups; ws: a device uint8
    tensor of at least toc_mgd_workspace_size(dev) bytes."""
    info = toc_dev_info_get(dev)
    if n_batches is None:
        n_batches = info["n_batches"] - b0
    if y.numel() < info["n_rows"] or y.element_size() != 4:
        raise TocError(TOC_EINVAL, "y must hold one float32 per row")
    if h.numel() != info["n_cols"] or h.element_size() != 4:
        raise TocError(TOC_EINVAL, "h must hold n_cols float32")
    _check(lib().toc_mgd_epoch_split(dev.handle, int(b0), int(n_batches), int(loss), float(lr),
                                     _ptr(y), _ptr(h), _ptr(ws), ws.numel() * ws.element_size(),
                                     _stream(stream)))


def toc_encode_device_workspace_size(n_batches, max_nnz):
    n = C.c_size_t()
    _check(lib().toc_encode_device_workspace_size(int(n_batches), int(max_nnz), C.byref(n)))
    return n.value


def toc_encode_device(n_rows, n_cols, rowptr, col, val, max_nnz, I_col, I_val, D_codes,
                      D_rowptr, counts, status, ws, stream=None):
    """Algorithm 1 on the device.  n_rows: host int32 array (one entry per batch);
    rowptr (int64), col (int32), val (float32): device tensors of the concatenated
    CSR; I_col, I_val, D_codes: device tensors of col.numel() entries; D_rowptr:
    device int64 tensor of sum(n_rows) + n_batches entries; counts: device int64
    tensor of 4 per batch; status: device int32 tensor of one per batch; ws: device
    tensor of toc_encode_device_workspace_size bytes."""
    n_rows = _arr(n_rows, np.int32)
    nb, nr = n_rows.size, int(n_rows.sum())
    nnz = col.numel()
    if rowptr.numel() != nr + 1 or rowptr.element_size() != 8:
        raise TocError(TOC_EINVAL, "rowptr must hold sum(n_rows) + 1 int64")
    if val.numel() != nnz or col.element_size() != 4 or val.element_size() != 4:
        raise TocError(TOC_EINVAL, "col and val must hold the same number of 4-byte entries")
    for t, name in ((I_col, "I_col"), (I_val, "I_val"), (D_codes, "D_codes")):
        if t.numel() < nnz or t.element_size() != 4:
            raise TocError(TOC_EINVAL, f"{name} must hold {nnz} 4-byte entries")
    if D_rowptr.numel() < nr + nb or D_rowptr.element_size() != 8:
        raise TocError(TOC_EINVAL, "D_rowptr must hold sum(n_rows) + n_batches int64")
    if counts.numel() < 4 * nb or counts.element_size() != 8:
        raise TocError(TOC_EINVAL, "counts must hold 4 int64 per batch")
    if status.numel() < nb or status.element_size() != 4:
        raise TocError(TOC_EINVAL, "status must hold one int32 per batch")
    _check(lib().toc_encode_device(nb, _ptr(n_rows), int(n_cols), _ptr(rowptr), _ptr(col),
                                   _ptr(val), nnz, int(max_nnz), _ptr(I_col), _ptr(I_val),
                                   _ptr(D_codes), _ptr(D_rowptr), _ptr(counts), _ptr(status),
                                   _ptr(ws), ws.numel() * ws.element_size() if ws is not None
                                   else 0, _stream(stream)))


def toc_mlp_workspace_size(dev, h1, h2, n_out):
    n = C.c_size_t()
    _check(lib().toc_mlp_workspace_size(dev.handle, int(h1), int(h2), int(n_out), C.byref(n)))
    return n.value


def toc_mlp_epoch(dev, params, labels, lr, ws, b0=0, n_batches=None, stream=None):
    """Neural-network MGD steps over batches b0 .. b0+n_batches-1 (default: all
    from b0).  params: dict of device float32 tensors W1 (m x h1), b1, W2 (h1 x
    h2), b2, W3 (h2 x n_out), b3, updated in place; labels: device int32 tensor of
    one label per row of the image; ws: device tensor of toc_mlp_workspace_size
    bytes."""
    info = toc_dev_info_get(dev)
    if n_batches is None:
        n_batches = info["n_batches"] - b0
    W1, W2, W3 = params["W1"], params["W2"], params["W3"]
    if W1.dim() != 2 or W2.dim() != 2 or W3.dim() != 2:
        raise TocError(TOC_EINVAL, "W1, W2, W3 must be matrices")
    m, h1 = W1.shape
    h2, n_out = W3.shape
    if m != info["n_cols"] or tuple(W2.shape) != (h1, h2):
        raise TocError(TOC_EINVAL, "parameter shapes do not chain m -> h1 -> h2 -> n_out")
    for name, t, n in (("W1", W1, m * h1), ("b1", params["b1"], h1), ("W2", W2, h1 * h2),
                       ("b2", params["b2"], h2), ("W3", W3, h2 * n_out),
                       ("b3", params["b3"], n_out)):
        if t.numel() != n or t.element_size() != 4 or not t.is_contiguous():
            raise TocError(TOC_EINVAL, f"{name} must be a contiguous float32 tensor of {n}")
    if labels.numel() < info["n_rows"] or labels.element_size() != 4:
        raise TocError(TOC_EINVAL, "labels must hold one int32 per row")
    _check(lib().toc_mlp_epoch(dev.handle, int(b0), int(n_batches), int(h1), int(h2),
                               int(n_out), _ptr(W1), _ptr(params["b1"]), _ptr(W2),
                               _ptr(params["b2"]), _ptr(W3), _ptr(params["b3"]), _ptr(labels),
                               float(lr), _ptr(ws), ws.numel() * ws.element_size(),
                               _stream(stream)))


def toc_level_workspace_size(n_batches, n_nodes):
    n = C.c_size_t()
    _check(lib().toc_level_workspace_size(int(n_batches), int(n_nodes), C.byref(n)))
    return n.value


def toc_level_build(blobs, blob_off, node_off, d_off, max_levels, cprime_status, parent, col,
                    val, depth, l_parent, l_col, l_val, l_depth, level, l_D, counts, status, ws,
                    stream=None):
    """blobs, blob_off, node_off and the cprime_* tensors as for toc_cprime_build;
    d_off: host int64 array of n_batches + 1 offsets into l_D; l_parent, l_col,
    l_val, l_depth: device tensors of node_off[-1] 4-byte entries; level: device
    int32/uint32 tensor of n_batches * (max_levels + 1); l_D: device tensor of
    d_off[-1] entries; counts: device int64 tensor of 2 per batch; status: device
    int32 tensor of one per batch; ws: toc_level_workspace_size bytes."""
    blob_off, node_off, d_off = (_arr(x, np.int64) for x in (blob_off, node_off, d_off))
    nb = blob_off.size - 1
    if node_off.size != nb + 1 or d_off.size != nb + 1:
        raise TocError(TOC_EINVAL, "offset arrays differ in length")
    n = int(node_off[-1])
    for t, name in ((parent, "parent"), (col, "col"), (val, "val"), (depth, "depth"),
                    (l_parent, "l_parent"), (l_col, "l_col"), (l_val, "l_val"),
                    (l_depth, "l_depth")):
        if t.numel() < n or t.element_size() != 4:
            raise TocError(TOC_EINVAL, f"{name} must hold {n} 4-byte entries")
    if level.numel() < nb * (int(max_levels) + 1) or level.element_size() != 4:
        raise TocError(TOC_EINVAL, "level must hold n_batches * (max_levels + 1) entries")
    if l_D.numel() < int(d_off[-1]) or l_D.element_size() != 4:
        raise TocError(TOC_EINVAL, "l_D shorter than d_off[-1]")
    if counts.numel() < 2 * nb or counts.element_size() != 8:
        raise TocError(TOC_EINVAL, "counts must hold 2 int64 per batch")
    for t, name in ((status, "status"), (cprime_status, "cprime_status")):
        if t.numel() < nb or t.element_size() != 4:
            raise TocError(TOC_EINVAL, f"{name} must hold one int32 per batch")
    if blobs.numel() < int(blob_off[-1]):
        raise TocError(TOC_EINVAL, "blobs shorter than blob_off[-1]")
    _check(lib().toc_level_build(_ptr(blobs), _ptr(blob_off), _ptr(node_off), _ptr(d_off), nb,
                                 int(max_levels), _ptr(cprime_status), _ptr(parent), _ptr(col),
                                 _ptr(val), _ptr(depth), _ptr(l_parent), _ptr(l_col),
                                 _ptr(l_val), _ptr(l_depth), _ptr(level), _ptr(l_D),
                                 _ptr(counts), _ptr(status), _ptr(ws),
                                 ws.numel() * ws.element_size() if ws is not None else 0,
                                 _stream(stream)))


def toc_level_right_mul(blobs, blob_off, node_off, d_off, row_off, max_levels, max_live,
                        level_status, counts, level, l_parent, l_col, l_val, l_D, w, r, status,
                        ws, stream=None):
    """A.w from toc_level_build's outputs (same launch arguments); row_off: host
    int64 array of n_batches + 1 row offsets into r; w: device float32 tensor of
    n_cols (its length is passed as n_cols: a key column at or above it gives the
    batch TOC_CPRIME_COLUMN); r: device float32 tensor of row_off[-1]; status:
    device int32 tensor of one per batch; ws: device tensor of at least
    32 (n_batches + 1) bytes."""
    blob_off, node_off, d_off, row_off = (_arr(x, np.int64)
                                          for x in (blob_off, node_off, d_off, row_off))
    nb = blob_off.size - 1
    if not (node_off.size == d_off.size == row_off.size == nb + 1):
        raise TocError(TOC_EINVAL, "offset arrays differ in length")
    if r.numel() < int(row_off[-1]) or r.element_size() != 4:
        raise TocError(TOC_EINVAL, "r must hold one float32 per row")
    if status.numel() < nb or status.element_size() != 4:
        raise TocError(TOC_EINVAL, "status must hold one int32 per batch")
    _check(lib().toc_level_right_mul(_ptr(blobs), _ptr(blob_off), _ptr(node_off), _ptr(d_off),
                                     _ptr(row_off), nb, int(w.numel()), int(max_levels),
                                     int(max_live),
                                     _ptr(level_status), _ptr(counts), _ptr(level),
                                     _ptr(l_parent), _ptr(l_col), _ptr(l_val), _ptr(l_D), _ptr(w),
                                     _ptr(r), _ptr(status), _ptr(ws),
                                     ws.numel() * ws.element_size(), _stream(stream)))
