"""ctypes binding of libvbq (C ABI declared in include/vbq.h).

Argument marshalling only: every step of the path -- quantizing and packing on
the host, decoding and multiplying on the GPU -- runs inside libvbq.  PyTorch
is used for device memory and streams.  If libvbq.so has not been built this
module raises on import; there is no fallback.
"""

import ctypes
import os

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libvbq.so")

if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is missing: build it with `python -m paper_2607_02893_amd.build` "
                      "(or __graft_entry__.build()); there is no fallback path")

try:
    # torch carries its own HIP runtime (SONAME libamdhip64.so.7).  Loading it
    # first makes libvbq bind to that same runtime, so device pointers and
    # stream handles from torch are valid in libvbq's calls.
    import torch as _torch  # noqa: F401
except ImportError:  # host-only use (packing) works with the system runtime
    _torch = None

_lib = ctypes.CDLL(LIB_PATH)


def hip_runtimes():
    """Paths of every HIP runtime library mapped into this process."""
    paths = set()
    try:
        with open("/proc/self/maps") as f:
            for line in f:
                if "libamdhip64" in line:
                    paths.add(os.path.realpath(line.split()[-1]))
    except OSError:
        pass
    return paths


if len(hip_runtimes()) > 1:
    raise ImportError(f"two HIP runtimes are loaded ({sorted(hip_runtimes())}); import torch before any other "
                      "HIP library so that libvbq binds to torch's runtime")

MAGIC = 0x31514256
LAYOUT_VERSION = 1
NSECTIONS = 10
MAX_M = 16
STATUS = {0: "VBQ_OK", 1: "VBQ_ERR_NULL", 2: "VBQ_ERR_SHAPE", 3: "VBQ_ERR_BITS", 4: "VBQ_ERR_CODE_RANGE",
          5: "VBQ_ERR_NONFINITE", 6: "VBQ_ERR_SCALE_RANGE", 7: "VBQ_ERR_BUFFER", 8: "VBQ_ERR_DESC",
          9: "VBQ_ERR_HIP", 10: "VBQ_ERR_UNSUPPORTED"}
# exported symbols, in the order include/vbq.h declares them
EXPORTS = ("vbq_status_string", "vbq_last_hip_error", "vbq_layout_version", "vbq_pack_size", "vbq_pack", "vbq_pack_codes",
           "vbq_desc_check", "vbq_gemv", "vbq_gemv_rows", "vbq_pack_row_buckets_size", "vbq_pack_row_buckets",
           "vbq_gemv_buckets", "vbq_gemm_small", "vbq_step_plan_bytes", "vbq_step_workspace_bytes",
           "vbq_step_plan", "vbq_step_run", "vbq_step_run_noalloc", "vbq_kernel_name", "vbq_gemv_buckets_kernel_name",
           "vbq_dequant",
           "vbq_qat_workspace_size", "vbq_qat_forward", "vbq_qat_logit_grad", "vbq_read_ceiling")
# vbq_desc.flags (call options)
Y_F16 = 1
ONE_WAVE_PER_UNIT = 2
MAX_BUCKETS = 4
QAT_MAX_GROUPS = 1 << 40
QAT_WSOFT_BF16 = 1
QAT_CANDIDATES = (1, 2, 4, 8)


class VbqDesc(ctypes.Structure):
    _fields_ = [("magic", ctypes.c_uint32), ("version", ctypes.c_uint32),
                ("N", ctypes.c_int64), ("K", ctypes.c_int64),
                ("group", ctypes.c_int32), ("tile_rows", ctypes.c_int32),
                ("chunk_groups", ctypes.c_int32), ("reserved0", ctypes.c_int32),
                ("n_tiles", ctypes.c_int64), ("n_chunks", ctypes.c_int64), ("n_units", ctypes.c_int64),
                ("n_entries", ctypes.c_int64 * 4),
                ("section_off", ctypes.c_uint64 * NSECTIONS), ("section_len", ctypes.c_uint64 * NSECTIONS),
                ("total_bytes", ctypes.c_uint64), ("flags", ctypes.c_uint32), ("reserved1", ctypes.c_uint32)]

    def info(self):
        """Plain-dict view (same keys as the oracle's pack info)."""
        return {"N": self.N, "K": self.K, "R": self.tile_rows, "C": self.chunk_groups,
                "T": self.n_tiles, "U": self.n_chunks, "units": self.n_units,
                "n_entries": list(self.n_entries), "section_off": list(self.section_off),
                "section_len": list(self.section_len), "total_bytes": self.total_bytes}


class VbqBucket(ctypes.Structure):
    _fields_ = [("bits", ctypes.c_int32), ("reserved", ctypes.c_int32), ("row_begin", ctypes.c_int64),
                ("n_rows", ctypes.c_int64), ("blob_offset", ctypes.c_uint64), ("desc", VbqDesc)]


class VbqStepGemv(ctypes.Structure):
    _fields_ = [("desc", ctypes.POINTER(VbqDesc)), ("blob", ctypes.c_void_p), ("x", ctypes.c_void_p),
                ("y", ctypes.c_void_p), ("rows", ctypes.c_void_p), ("y_len", ctypes.c_int64)]


class VbqPackOpts(ctypes.Structure):
    _fields_ = [("tile_rows", ctypes.c_int32), ("chunk_groups", ctypes.c_int32),
                ("flags", ctypes.c_uint32), ("n_threads", ctypes.c_uint32)]


_P = ctypes.c_void_p
_lib.vbq_status_string.restype = ctypes.c_char_p
_lib.vbq_status_string.argtypes = [ctypes.c_int]
_lib.vbq_last_hip_error.restype = ctypes.c_char_p
_lib.vbq_last_hip_error.argtypes = []
_lib.vbq_layout_version.restype = ctypes.c_uint32
_lib.vbq_layout_version.argtypes = []
_lib.vbq_pack_size.restype = ctypes.c_int
_lib.vbq_pack_size.argtypes = [ctypes.c_int64, ctypes.c_int64, _P, ctypes.POINTER(VbqPackOpts),
                               ctypes.POINTER(ctypes.c_size_t), ctypes.POINTER(VbqDesc)]
_lib.vbq_pack.restype = ctypes.c_int
_lib.vbq_pack.argtypes = [ctypes.c_int64, ctypes.c_int64, _P, _P, ctypes.POINTER(VbqPackOpts), _P,
                          ctypes.c_size_t, ctypes.POINTER(VbqDesc)]
_lib.vbq_pack_codes.restype = ctypes.c_int
_lib.vbq_pack_codes.argtypes = [ctypes.c_int64, ctypes.c_int64, _P, _P, _P, ctypes.POINTER(VbqPackOpts), _P,
                                ctypes.c_size_t, ctypes.POINTER(VbqDesc)]
_lib.vbq_desc_check.restype = ctypes.c_int
_lib.vbq_desc_check.argtypes = [ctypes.POINTER(VbqDesc)]
_lib.vbq_gemv.restype = ctypes.c_int
_lib.vbq_gemv.argtypes = [ctypes.POINTER(VbqDesc), _P, _P, _P, _P]
_lib.vbq_gemv_rows.restype = ctypes.c_int
_lib.vbq_gemv_rows.argtypes = [ctypes.POINTER(VbqDesc), _P, _P, _P, ctypes.c_int64, _P, _P]
_lib.vbq_pack_row_buckets_size.restype = ctypes.c_int
_lib.vbq_pack_row_buckets_size.argtypes = [ctypes.c_int64, ctypes.c_int64, _P, ctypes.POINTER(VbqPackOpts),
                                           ctypes.POINTER(ctypes.c_size_t), ctypes.POINTER(ctypes.c_int32)]
_lib.vbq_pack_row_buckets.restype = ctypes.c_int
_lib.vbq_pack_row_buckets.argtypes = [ctypes.c_int64, ctypes.c_int64, _P, _P, _P, ctypes.POINTER(VbqPackOpts), _P,
                                      ctypes.c_size_t, ctypes.POINTER(VbqBucket), ctypes.POINTER(ctypes.c_int32), _P]
_lib.vbq_gemv_buckets.restype = ctypes.c_int
_lib.vbq_gemv_buckets.argtypes = [ctypes.POINTER(VbqBucket), ctypes.c_int32, _P, _P, _P, _P, ctypes.c_int64, _P]
_lib.vbq_gemm_small.restype = ctypes.c_int
_lib.vbq_gemm_small.argtypes = [ctypes.POINTER(VbqDesc), _P, ctypes.c_int64, _P, ctypes.c_int64, _P,
                                ctypes.c_int64, _P]
_lib.vbq_step_plan_bytes.restype = ctypes.c_int
_lib.vbq_step_plan_bytes.argtypes = [ctypes.c_int32, ctypes.POINTER(ctypes.c_size_t)]
_lib.vbq_step_workspace_bytes.restype = ctypes.c_int
_lib.vbq_step_workspace_bytes.argtypes = [ctypes.c_int32, ctypes.POINTER(ctypes.c_size_t)]
_lib.vbq_step_plan.restype = ctypes.c_int
_lib.vbq_step_plan.argtypes = [ctypes.POINTER(VbqStepGemv), ctypes.c_int32, _P, ctypes.c_size_t]
_lib.vbq_step_run.restype = ctypes.c_int
_lib.vbq_step_run.argtypes = [_P, ctypes.c_int32, _P, ctypes.c_size_t, ctypes.c_uint32, _P]
_lib.vbq_step_run_noalloc.restype = ctypes.c_int
_lib.vbq_step_run_noalloc.argtypes = [_P, ctypes.c_int32, ctypes.c_uint32, _P, _P]
_lib.vbq_kernel_name.restype = ctypes.c_char_p
_lib.vbq_kernel_name.argtypes = [ctypes.POINTER(VbqDesc), ctypes.c_int64]
_lib.vbq_gemv_buckets_kernel_name.restype = ctypes.c_char_p
_lib.vbq_gemv_buckets_kernel_name.argtypes = [ctypes.POINTER(VbqBucket), ctypes.c_int32]
_lib.vbq_read_ceiling.restype = ctypes.c_int
_lib.vbq_read_ceiling.argtypes = [_P, ctypes.c_size_t, ctypes.c_uint32, _P, _P]
_lib.vbq_dequant.restype = ctypes.c_int
_lib.vbq_dequant.argtypes = [ctypes.POINTER(VbqDesc), _P, _P, _P]
_lib.vbq_qat_workspace_size.restype = ctypes.c_int
_lib.vbq_qat_workspace_size.argtypes = [ctypes.c_int64, ctypes.POINTER(ctypes.c_size_t)]
_lib.vbq_qat_forward.restype = ctypes.c_int
_lib.vbq_qat_forward.argtypes = [ctypes.c_int64, _P, _P, _P, ctypes.c_float, ctypes.c_uint32, _P, _P, _P, _P, _P,
                                 ctypes.c_size_t, _P]
_lib.vbq_qat_logit_grad.restype = ctypes.c_int
_lib.vbq_qat_logit_grad.argtypes = [ctypes.c_int64, _P, _P, _P, ctypes.c_float, ctypes.c_float, ctypes.c_int64, _P, _P]


class VbqError(RuntimeError):
    def __init__(self, status, where):
        self.status = status
        msg = _lib.vbq_status_string(status).decode()
        if status == 9:
            msg += f": {_lib.vbq_last_hip_error().decode()}"
        super().__init__(f"{where}: {STATUS.get(status, status)} ({msg})")


def _check(status, where):
    if status != 0:
        raise VbqError(status, where)


def status_string(status):
    return _lib.vbq_status_string(status).decode()


def layout_version():
    return int(_lib.vbq_layout_version())


def _opts(tile_rows=0, chunk_groups=0, n_threads=0):
    return VbqPackOpts(tile_rows, chunk_groups, 0, n_threads)


def _ptr(a):
    return a.ctypes.data_as(ctypes.c_void_p) if a is not None else None


def pack_size(bits, K, tile_rows=0, chunk_groups=0):
    bits = np.ascontiguousarray(bits, dtype=np.uint8)
    nbytes = ctypes.c_size_t(0)
    d = VbqDesc()
    o = _opts(tile_rows, chunk_groups)
    _check(_lib.vbq_pack_size(bits.shape[0], K, _ptr(bits), ctypes.byref(o), ctypes.byref(nbytes),
                              ctypes.byref(d)), "vbq_pack_size")
    return nbytes.value, d


def _blob(nbytes):
    # 256-byte aligned host buffer
    raw = np.zeros(nbytes + 256, dtype=np.uint8)
    off = (-raw.ctypes.data) % 256
    return raw[off:off + nbytes]


def pack(W, bits, tile_rows=0, chunk_groups=0, n_threads=0):
    """Quantize float32 W[N][K] with bit map bits[N][K/64] and pack it (host)."""
    W = np.ascontiguousarray(W, dtype=np.float32)
    bits = np.ascontiguousarray(bits, dtype=np.uint8)
    N, K = W.shape
    nbytes, _ = pack_size(bits, K, tile_rows, chunk_groups)
    blob = _blob(nbytes)
    d = VbqDesc()
    o = _opts(tile_rows, chunk_groups, n_threads)
    _check(_lib.vbq_pack(N, K, _ptr(W), _ptr(bits), ctypes.byref(o), _ptr(blob), nbytes, ctypes.byref(d)),
           "vbq_pack")
    return blob, d


def pack_codes(q, scales, bits, tile_rows=0, chunk_groups=0, n_threads=0):
    """Pack levels q int8[N][K], fp16 scale bits uint16[N][K/64] and bits uint8[N][K/64] (host)."""
    q = np.ascontiguousarray(q, dtype=np.int8)
    scales = np.ascontiguousarray(scales, dtype=np.uint16)
    bits = np.ascontiguousarray(bits, dtype=np.uint8)
    N, K = q.shape
    nbytes, _ = pack_size(bits, K, tile_rows, chunk_groups)
    blob = _blob(nbytes)
    d = VbqDesc()
    o = _opts(tile_rows, chunk_groups, n_threads)
    _check(_lib.vbq_pack_codes(N, K, _ptr(q), _ptr(scales), _ptr(bits), ctypes.byref(o), _ptr(blob), nbytes,
                               ctypes.byref(d)), "vbq_pack_codes")
    return blob, d


def pack_row_buckets_raw(q, scales, row_bits, tile_rows=0, chunk_groups=0, n_threads=0):
    """vbq_pack_row_buckets: (blob, [VbqBucket], row_index int32[N]) for levels
    q int8[N][K], fp16 scale bits uint16[N][K/64] and one width per row."""
    q = np.ascontiguousarray(q, dtype=np.int8)
    scales = np.ascontiguousarray(scales, dtype=np.uint16)
    row_bits = np.ascontiguousarray(row_bits, dtype=np.uint8)
    N, K = q.shape
    o = _opts(tile_rows, chunk_groups, n_threads)
    nbytes = ctypes.c_size_t(0)
    nb = ctypes.c_int32(0)
    _check(_lib.vbq_pack_row_buckets_size(N, K, _ptr(row_bits), ctypes.byref(o), ctypes.byref(nbytes),
                                          ctypes.byref(nb)), "vbq_pack_row_buckets_size")
    blob = _blob(nbytes.value)
    bk = (VbqBucket * MAX_BUCKETS)()
    row_index = np.empty(N, dtype=np.int32)
    _check(_lib.vbq_pack_row_buckets(N, K, _ptr(q), _ptr(scales), _ptr(row_bits), ctypes.byref(o), _ptr(blob),
                                     nbytes.value, bk, ctypes.byref(nb), _ptr(row_index)), "vbq_pack_row_buckets")
    return blob, [bk[i] for i in range(nb.value)], row_index


def pack_row_buckets(q, scales, bits, tile_rows=0, chunk_groups=0, n_threads=0):
    """Pack a matrix whose rows each have one width (a recipe head: paper section
    4, frequency-tiered rows; section 6, stored as frequency-grouped row buckets)
    as one packed matrix per width (vbq_pack_row_buckets).  Returns
    [(width, rows, blob, desc)] in increasing width, rows the int32 output rows
    of the bucket's members in order and blob that bucket's bytes.  Each bucket
    has one width, so it carries no width map."""
    bits = np.ascontiguousarray(bits, dtype=np.uint8)
    w = bits[:, 0]
    if not np.array_equal(bits, np.repeat(w[:, None], bits.shape[1], axis=1)):
        raise ValueError("row buckets need one width per row")
    blob, bk, row_index = pack_row_buckets_raw(q, scales, w, tile_rows, chunk_groups, n_threads)
    out = []
    for b in bk:
        off, n = int(b.blob_offset), int(b.n_rows)
        d = VbqDesc.from_buffer_copy(b.desc)
        out.append((int(b.bits), row_index[b.row_begin:b.row_begin + n].copy(),
                    blob[off:off + int(d.total_bytes)], d))
    return RowBuckets(out, blob, bk, row_index)


class RowBuckets(list):
    """pack_row_buckets' result: [(width, rows, blob, desc)] per bucket, plus the
    whole blob, the bucket table and the row index as vbq_pack_row_buckets wrote
    them (what vbq_gemv_buckets takes)."""

    def __init__(self, items, blob, buckets, row_index):
        super().__init__(items)
        self.blob, self.buckets, self.row_index = blob, buckets, row_index


def buckets_kernel_name(buckets):
    """vbq_gemv_buckets_kernel_name for a list of VbqBucket."""
    table = (VbqBucket * max(1, len(buckets)))(*buckets)
    return _lib.vbq_gemv_buckets_kernel_name(table, len(buckets)).decode()


def desc_check(d):
    return _lib.vbq_desc_check(ctypes.byref(d))


class Step:
    """A decode step run as one launch (vbq_step_run): a sequence of GEMVs, GEMV
    i reading its x only after every earlier GEMV has written its y.

    gemvs: list of (desc, blob_ptr, x_ptr, y_ptr, rows_ptr or 0, y_len) on one
    device; the plan and the workspace are allocated here with torch (device
    memory), and the host plan image is built by vbq_step_plan."""

    def __init__(self, gemvs, device="cuda"):
        import torch
        n = len(gemvs)
        self.n = n
        self._descs = [VbqDesc.from_buffer_copy(g[0]) for g in gemvs]  # kept alive for the plan call
        arr = (VbqStepGemv * n)()
        for i, (g, d) in enumerate(zip(gemvs, self._descs)):
            arr[i] = VbqStepGemv(ctypes.pointer(d), g[1], g[2], g[3], g[4] or None, int(g[5]))
        pb, wb = ctypes.c_size_t(0), ctypes.c_size_t(0)
        _check(_lib.vbq_step_plan_bytes(n, ctypes.byref(pb)), "vbq_step_plan_bytes")
        _check(_lib.vbq_step_workspace_bytes(n, ctypes.byref(wb)), "vbq_step_workspace_bytes")
        host = np.zeros(pb.value, dtype=np.uint8)
        _check(_lib.vbq_step_plan(arr, n, _ptr(host), pb.value), "vbq_step_plan")
        self.plan = torch.from_numpy(host).to(device)
        self.workspace = torch.zeros(wb.value // 4, dtype=torch.int32, device=device)

    def run(self, stream=None, spin_limit=0):
        return _lib.vbq_step_run(ctypes.c_void_p(self.plan.data_ptr()), self.n,
                                 ctypes.c_void_p(self.workspace.data_ptr()), self.workspace.numel() * 4,
                                 int(spin_limit), _stream_handle(stream))

    def run_noalloc(self, status=None, stream=None, spin_limit=0):
        """vbq_step_run_noalloc (the library's own scratch); status: an optional
        int32 device tensor of one element that receives the status word."""
        return _lib.vbq_step_run_noalloc(ctypes.c_void_p(self.plan.data_ptr()), self.n, int(spin_limit),
                                         ctypes.c_void_p(status.data_ptr()) if status is not None else None,
                                         _stream_handle(stream))

    def status(self):
        """The status word (0 after a complete run); synchronizes."""
        return int(self.workspace[-1].item())


def kernel_name(d, M=1):
    """Name of the kernel a product with M activation rows launches on this matrix."""
    return _lib.vbq_kernel_name(ctypes.byref(d), int(M)).decode()


def raw_read_ceiling(src_ptr, nbytes, blocks, sink_ptr, stream_ptr):
    """vbq_read_ceiling on raw device addresses."""
    return _lib.vbq_read_ceiling(ctypes.c_void_p(src_ptr), int(nbytes), int(blocks), ctypes.c_void_p(sink_ptr),
                                 ctypes.c_void_p(stream_ptr))


# ------------------------------------------------------------------ device side

def _stream_handle(stream):
    import torch
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _need(t, name, dtype, numel=None, device=None, min_numel=None):
    """A device tensor the kernels may read or write: on a GPU (a host pointer
    would fault in a kernel), of the given dtype, contiguous and of the given
    size (exact, or at least min_numel), on `device` when given."""
    if t is None or not getattr(t, "is_cuda", False):
        raise ValueError(f"{name} must be a GPU tensor")
    if t.dtype != dtype or not t.is_contiguous():
        raise ValueError(f"{name} must be a contiguous {dtype} tensor")
    if numel is not None and t.numel() != numel:
        raise ValueError(f"{name} must have {numel} elements, not {t.numel()}")
    if min_numel is not None and t.numel() < min_numel:
        raise ValueError(f"{name} must have at least {min_numel} elements")
    if device is not None and t.device != device:
        raise ValueError(f"{name} is on {t.device}, expected {device}")
    return t


class PackedMatrix:
    """A packed matrix resident in device memory (torch uint8 tensor) plus its descriptor."""

    def __init__(self, blob, desc, device="cuda"):
        import torch
        self.desc = desc
        self.N, self.K = desc.N, desc.K
        t = torch.from_numpy(np.asarray(blob, dtype=np.uint8))
        # torch's caching allocator returns 256-byte aligned blocks
        self.blob = t.to(device)
        if self.blob.data_ptr() % 256:
            raise VbqError(7, "PackedMatrix")

    @classmethod
    def on_device(cls, blob, desc):
        """A packed matrix whose bytes are already in device memory (a uint8 tensor,
        e.g. one bucket's slice of a bucketed blob), 256-byte aligned."""
        self = cls.__new__(cls)
        self.desc = desc
        self.N, self.K = desc.N, desc.K
        self.blob = blob
        if blob.data_ptr() % 256:
            raise VbqError(7, "PackedMatrix")
        return self

    @property
    def nbytes(self):
        return int(self.desc.total_bytes)

    def call_desc(self, y_dtype=None, one_wave_per_unit=False):
        """A copy of the descriptor with the call options set: fp16 output
        (y_dtype torch.float16) and one wave per unit."""
        import torch
        d = VbqDesc.from_buffer_copy(self.desc)
        d.flags = (Y_F16 if y_dtype == torch.float16 else 0) | (ONE_WAVE_PER_UNIT if one_wave_per_unit else 0)
        return d

    def gemv(self, x, y=None, stream=None, y_dtype=None, one_wave_per_unit=False):
        """y[N] = w_hat @ x, x a contiguous fp16 device tensor of length K; y float32,
        or float16 (VBQ_Y_F16: the fp32 result rounded to nearest even) when
        y_dtype or the given y says so."""
        import torch
        dev = self.blob.device
        _need(x, "x", torch.float16, self.K, dev)
        y_dtype = (y.dtype if y is not None else torch.float32) if y_dtype is None else y_dtype
        if y_dtype not in (torch.float32, torch.float16):
            raise ValueError("y must be float32 or float16")
        if y is None:
            y = torch.empty(self.N, dtype=y_dtype, device=dev)
        _need(y, "y", y_dtype, self.N, dev)
        d = self.call_desc(y_dtype, one_wave_per_unit)
        _check(_lib.vbq_gemv(ctypes.byref(d), ctypes.c_void_p(self.blob.data_ptr()),
                             ctypes.c_void_p(x.data_ptr()), ctypes.c_void_p(y.data_ptr()),
                             _stream_handle(stream)), "vbq_gemv")
        return y

    def gemv_rows(self, x, y, rows, stream=None):
        """y[rows[n]] = (w_hat @ x)[n] for every n (indices outside y are not written): one row
        bucket of a bucketed matrix.  y: float32 (or float16) device tensor; rows: int32 device tensor
        of length N."""
        import torch
        dev = self.blob.device
        _need(x, "x", torch.float16, self.K, dev)
        if y.dtype not in (torch.float32, torch.float16):
            raise ValueError("y must be float32 or float16")
        _need(y, "y", y.dtype, None, dev)
        _need(rows, "rows", torch.int32, self.N, dev)
        d = self.call_desc(y.dtype)
        _check(_lib.vbq_gemv_rows(ctypes.byref(d), ctypes.c_void_p(self.blob.data_ptr()),
                                  ctypes.c_void_p(x.data_ptr()), ctypes.c_void_p(y.data_ptr()), y.numel(),
                                  ctypes.c_void_p(rows.data_ptr()), _stream_handle(stream)), "vbq_gemv_rows")
        return y

    def gemm_small(self, X, Y=None, stream=None, y_dtype=None, one_wave_per_unit=False):
        """Y[M][N] = X @ w_hat^T for an fp16 device tensor X[M][K], M <= 16 (rows may be
        padded: X.stride(0) >= K); Y float32, or float16 when y_dtype or the given Y says so."""
        import torch
        dev = self.blob.device
        if not getattr(X, "is_cuda", False) or X.device != dev:
            raise ValueError(f"X must be a GPU tensor on {dev}")
        if X.dtype != torch.float16 or X.dim() != 2 or X.shape[1] != self.K or X.stride(1) != 1:
            raise ValueError("X must be a float16 [M, K] tensor with unit column stride")
        M = X.shape[0]
        y_dtype = (Y.dtype if Y is not None else torch.float32) if y_dtype is None else y_dtype
        if Y is None:
            Y = torch.empty((M, self.N), dtype=y_dtype, device=dev)
        if (not getattr(Y, "is_cuda", False) or Y.device != dev or Y.dtype != y_dtype
                or y_dtype not in (torch.float32, torch.float16) or Y.dim() != 2
                or Y.shape[0] != M or Y.shape[1] != self.N or Y.stride(1) != 1):
            raise ValueError(f"Y must be a float32/float16 [M, N] GPU tensor on {dev} with unit column stride")
        d = self.call_desc(y_dtype, one_wave_per_unit)
        _check(_lib.vbq_gemm_small(ctypes.byref(d), ctypes.c_void_p(self.blob.data_ptr()), M,
                                   ctypes.c_void_p(X.data_ptr()), X.stride(0), ctypes.c_void_p(Y.data_ptr()),
                                   Y.stride(0), _stream_handle(stream)), "vbq_gemm_small")
        return Y

    def dequant(self, W=None, stream=None):
        """w_hat as a float32 [N, K] device tensor (exact)."""
        import torch
        if W is None:
            W = torch.empty((self.N, self.K), dtype=torch.float32, device=self.blob.device)
        _need(W, "W", torch.float32, self.N * self.K, self.blob.device)
        _check(_lib.vbq_dequant(ctypes.byref(self.desc), ctypes.c_void_p(self.blob.data_ptr()),
                                ctypes.c_void_p(W.data_ptr()), _stream_handle(stream)), "vbq_dequant")
        return W


class BucketedMatrix:
    """A row-bucketed matrix in device memory: one PackedMatrix per width and
    the output rows of its members (see pack_row_buckets).  From a RowBuckets
    the whole blob and row index go to the device as one buffer each, and gemv
    is one vbq_gemv_buckets call."""

    def __init__(self, buckets, N, K, device="cuda"):
        import torch
        self.N, self.K = N, K
        self.table = None
        if isinstance(buckets, RowBuckets):
            self.blob = torch.from_numpy(np.asarray(buckets.blob, dtype=np.uint8)).to(device)
            self.row_index = torch.from_numpy(np.ascontiguousarray(buckets.row_index)).to(device)
            self.table = (VbqBucket * MAX_BUCKETS)(*buckets.buckets)
            self.n_buckets = len(buckets.buckets)
            self.parts = []
            for (b, _, _, d), bk in zip(buckets, buckets.buckets):
                off, r0, n = int(bk.blob_offset), int(bk.row_begin), int(bk.n_rows)
                part = PackedMatrix.on_device(self.blob[off:off + int(d.total_bytes)], d)
                self.parts.append((b, part, self.row_index[r0:r0 + n]))
        else:
            self.parts = [(b, PackedMatrix(blob, d, device), torch.from_numpy(rows).to(device))
                          for b, rows, blob, d in buckets]
        if sum(p[1].N for p in self.parts) != N:
            raise ValueError("the buckets must hold every row once")

    @property
    def nbytes(self):
        return sum(p[1].nbytes for p in self.parts)

    def kernel_name(self):
        """What gemv launches (vbq_gemv_buckets_kernel_name), or "per bucket"."""
        if self.table is None:
            return "per bucket"
        return _lib.vbq_gemv_buckets_kernel_name(self.table, self.n_buckets).decode()

    def call_table(self, y_dtype):
        """A copy of the bucket table with the fp16-output option set or cleared."""
        import torch
        t = (VbqBucket * MAX_BUCKETS)()
        ctypes.memmove(t, self.table, ctypes.sizeof(t))
        for i in range(self.n_buckets):
            t[i].desc.flags = Y_F16 if y_dtype == torch.float16 else 0
        return t

    def gemv(self, x, y=None, stream=None):
        """y[N] = w_hat @ x; y float32 (or a given float16 tensor).  One
        vbq_gemv_buckets call (from a RowBuckets), else one vbq_gemv_rows per
        bucket, on one stream."""
        import torch
        dev = self.parts[0][1].blob.device
        if y is None:
            y = torch.empty(self.N, dtype=torch.float32, device=dev)
        if y.dtype not in (torch.float32, torch.float16):
            raise ValueError("y must be float32 or float16")
        _need(y, "y", y.dtype, self.N, dev)
        if self.table is not None:
            _need(x, "x", torch.float16, self.K, dev)
            _check(_lib.vbq_gemv_buckets(self.call_table(y.dtype), self.n_buckets,
                                         ctypes.c_void_p(self.blob.data_ptr()),
                                         ctypes.c_void_p(self.row_index.data_ptr()), ctypes.c_void_p(x.data_ptr()),
                                         ctypes.c_void_p(y.data_ptr()), y.numel(), _stream_handle(stream)),
                   "vbq_gemv_buckets")
            return y
        for _, Wp, rows in self.parts:
            Wp.gemv_rows(x, y, rows, stream)
        return y


def raw_gemv_buckets(table, n_buckets, blob_ptr, row_index_ptr, x_ptr, y_ptr, y_len, stream_ptr):
    """vbq_gemv_buckets with raw device addresses (a ctypes VbqBucket array)."""
    return _lib.vbq_gemv_buckets(table, n_buckets, ctypes.c_void_p(blob_ptr), ctypes.c_void_p(row_index_ptr),
                                 ctypes.c_void_p(x_ptr), ctypes.c_void_p(y_ptr), y_len, ctypes.c_void_p(stream_ptr))


# ------------------------------------------------- differentiable bit selection

def qat_workspace_size(n_groups):
    """Device workspace bytes vbq_qat_forward needs for bbar over n_groups groups."""
    nbytes = ctypes.c_size_t(0)
    _check(_lib.vbq_qat_workspace_size(int(n_groups), ctypes.byref(nbytes)), "vbq_qat_workspace_size")
    return nbytes.value


def _dev_ptr(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else None


def qat_forward(W, logits, noise, tau, w_soft=None, pi=True, hard_bits=True, bbar=True, workspace=None,
                stream=None, w_soft_dtype=None):
    """Forward pass of the selection path (paper section 3.2, Algorithm 1) on device tensors.

    W: contiguous float32 device tensor whose numel is a multiple of 64 (its
    groups are consecutive runs of 64; a row-major [N, K] matrix with K % 64 == 0
    qualifies).  logits / noise: contiguous float32 [n_groups, 4] (any shape of
    that size); noise may be None.  pi / hard_bits / bbar: True to allocate the
    output, a tensor to write into, or False/None to skip it.  w_soft is float32,
    or bfloat16 (each value rounded to nearest even) when w_soft_dtype or the
    given w_soft tensor says so.  Returns
    (w_soft, pi, hard_bits, bbar) with bbar a float64 device tensor of one
    element (None where skipped).
    """
    import torch
    _need(W, "W", torch.float32)
    if W.numel() % 64:
        raise ValueError("W must have a multiple of 64 elements")
    n = W.numel() // 64
    dev = W.device
    _need(logits, "logits", torch.float32, 4 * n, dev)
    if noise is not None:
        _need(noise, "noise", torch.float32, 4 * n, dev)
    if w_soft_dtype is None:
        w_soft_dtype = torch.float32 if w_soft is None else w_soft.dtype
    if w_soft_dtype not in (torch.float32, torch.bfloat16):
        raise ValueError("w_soft must be float32 or bfloat16")
    if w_soft is None:
        w_soft = torch.empty(W.shape, dtype=w_soft_dtype, device=dev)
    _need(w_soft, "w_soft", w_soft_dtype, W.numel(), dev)
    flags = QAT_WSOFT_BF16 if w_soft_dtype == torch.bfloat16 else 0
    if pi is True:
        pi = torch.empty((n, 4), dtype=torch.float32, device=dev)
    if hard_bits is True:
        hard_bits = torch.empty(n, dtype=torch.uint8, device=dev)
    if bbar is True:
        bbar = torch.empty(1, dtype=torch.float64, device=dev)
    pi = pi if pi is not False else None
    hard_bits = hard_bits if hard_bits is not False else None
    bbar = bbar if bbar is not False else None
    if pi is not None:
        _need(pi, "pi", torch.float32, 4 * n, dev)
    if hard_bits is not None:
        _need(hard_bits, "hard_bits", torch.uint8, n, dev)
    ws_bytes = 0
    if bbar is not None:
        _need(bbar, "bbar", torch.float64, None, dev, min_numel=1)
        ws_bytes = qat_workspace_size(n)
        if workspace is None:
            workspace = torch.empty(max(ws_bytes, 8), dtype=torch.uint8, device=dev)
        _need(workspace, "workspace", workspace.dtype, None, dev)
        ws_bytes = workspace.numel() * workspace.element_size()
    _check(_lib.vbq_qat_forward(n, _dev_ptr(W), _dev_ptr(logits), _dev_ptr(noise), float(tau), flags, _dev_ptr(w_soft),
                                _dev_ptr(pi), _dev_ptr(hard_bits), _dev_ptr(bbar), _dev_ptr(workspace), ws_bytes,
                                _stream_handle(stream)), "vbq_qat_forward")
    return w_soft, pi, hard_bits, bbar


def qat_logit_grad(W, grad, pi, tau, lam, n_bbar=None, dlogits=None, stream=None):
    """Logit-step gradient (paper section 3.3, Algorithm 1) on device tensors.

    W, grad: contiguous float32 tensors of n_groups*64 elements (the forward's
    weights and dL_CE/dw_soft); pi: the forward's float32 [n_groups, 4];
    n_bbar: the n of bbar (default n_groups).  Returns dL/dlogits, float32
    [n_groups, 4].
    """
    import torch
    _need(W, "W", torch.float32)
    if W.numel() % 64:
        raise ValueError("W must have a multiple of 64 elements")
    n = W.numel() // 64
    dev = W.device
    _need(grad, "grad", torch.float32, W.numel(), dev)
    _need(pi, "pi", torch.float32, 4 * n, dev)
    if dlogits is None:
        dlogits = torch.empty((n, 4), dtype=torch.float32, device=dev)
    _need(dlogits, "dlogits", torch.float32, 4 * n, dev)
    _check(_lib.vbq_qat_logit_grad(n, _dev_ptr(W), _dev_ptr(grad), _dev_ptr(pi), float(tau), float(lam),
                                   int(n if n_bbar is None else n_bbar), _dev_ptr(dlogits), _stream_handle(stream)),
           "vbq_qat_logit_grad")
    return dlogits


def raw_qat_logit_grad(n_groups, W_ptr, grad_ptr, pi_ptr, tau, lam, n_bbar, d_ptr, stream_ptr):
    """vbq_qat_logit_grad on raw device addresses (0 for NULL)."""
    v = lambda p: ctypes.c_void_p(p) if p else None  # noqa: E731
    return _lib.vbq_qat_logit_grad(int(n_groups), v(W_ptr), v(grad_ptr), v(pi_ptr), float(tau), float(lam),
                                   int(n_bbar), v(d_ptr), v(stream_ptr))


def raw_qat_forward(n_groups, W_ptr, logits_ptr, noise_ptr, tau, w_soft_ptr, pi_ptr, hard_ptr, bbar_ptr,
                    ws_ptr, ws_bytes, stream_ptr, flags=0):
    """vbq_qat_forward on raw device addresses (0 for NULL)."""
    v = lambda p: ctypes.c_void_p(p) if p else None  # noqa: E731
    return _lib.vbq_qat_forward(int(n_groups), v(W_ptr), v(logits_ptr), v(noise_ptr), float(tau), int(flags),
                                v(w_soft_ptr),
                                v(pi_ptr), v(hard_ptr), v(bbar_ptr), v(ws_ptr), int(ws_bytes), v(stream_ptr))


def raw_gemv(desc, blob_ptr, x_ptr, y_ptr, stream_ptr):
    """vbq_gemv on raw device addresses (no checks beyond the library's own)."""
    return _lib.vbq_gemv(ctypes.byref(desc), ctypes.c_void_p(blob_ptr), ctypes.c_void_p(x_ptr),
                         ctypes.c_void_p(y_ptr), ctypes.c_void_p(stream_ptr))


def raw_gemv_rows(desc, blob_ptr, x_ptr, y_ptr, y_len, rows_ptr, stream_ptr):
    """vbq_gemv_rows on raw device addresses."""
    return _lib.vbq_gemv_rows(ctypes.byref(desc), ctypes.c_void_p(blob_ptr), ctypes.c_void_p(x_ptr),
                              ctypes.c_void_p(y_ptr), y_len, ctypes.c_void_p(rows_ptr), ctypes.c_void_p(stream_ptr))


def raw_gemm_small(desc, blob_ptr, M, X_ptr, ldx, Y_ptr, ldy, stream_ptr):
    return _lib.vbq_gemm_small(ctypes.byref(desc), ctypes.c_void_p(blob_ptr), M, ctypes.c_void_p(X_ptr), ldx,
                               ctypes.c_void_p(Y_ptr), ldy, ctypes.c_void_p(stream_ptr))


def lib():
    """The loaded ctypes library (for symbol checks)."""
    return _lib
