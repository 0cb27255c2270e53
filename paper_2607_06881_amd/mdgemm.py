"""Python binding of ``libmdgemm.so`` (C ABI in ``include/mdgemm.h``).

Argument marshalling only: every step of the product runs in the library's
HIP kernels.  PyTorch provides device memory (tensors, the workspace) and the
stream (``torch.cuda.current_stream()``).  The functions carry the names of the
C entry points.  If the library is missing this module raises: there is no
fallback path.
"""

from __future__ import annotations

import ctypes
import os
from typing import Optional

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libmdgemm.so")

MDGEMM_OK = 0
MDGEMM_EINVAL = -1
MDGEMM_EEXACT = -2
MDGEMM_ENOMEM = -3
MDGEMM_EHIP = -4
MDGEMM_EWORKSPACE = -5
MDGEMM_ENONFINITE = -6

MDGEMM_CHECK_FINITE = 1
MDGEMM_SYNC = 2
MDGEMM_TIME_STAGES = 4
MDGEMM_KARATSUBA = 8
MDGEMM_KARATSUBA_MIN_TERMS = 16
MDGEMM_INT8 = 32
MDGEMM_STAGED = 64
MDGEMM_GROUP_SIGN = 128
MDGEMM_GROUP_EXPONENT = 256
MDGEMM_SCHEDULE_INFO = 12
MDGEMM_LAYOUT_INFO = 12
MDGEMM_NOALLOC_MAX_BYTES = 64 << 20

MDGEMM_CUTOFF_DEFAULT = -1
MDGEMM_CUTOFF_ALL = -2
MDGEMM_MAX_LIMBS = 16
MDGEMM_MAX_SLICES = 68
MDGEMM_MAX_LEVELS = 135
MDGEMM_SLICE_BITS = 13
MDGEMM_MAX_SLICE_BITS = 26
MDGEMM_MAX_DIGIT_BITS = 908
MDGEMM_SLICE_BITS_AUTO = -1
MDGEMM_Z_WORDS = 28
PANEL_K = 16  # level-GEMM panels: k rounded up to 16,
PANEL_MN = 128  # m and n rounded up to 128
PANEL_K32 = 32  # FP32 panels inside mdgemm_ex: k rounded up to 32


def panel_k(k: int) -> int:
    return (k + PANEL_K - 1) // PANEL_K * PANEL_K


def panel_k32(k: int) -> int:
    return (k + PANEL_K32 - 1) // PANEL_K32 * PANEL_K32


def panel_mn(x: int) -> int:
    return (x + PANEL_MN - 1) // PANEL_MN * PANEL_MN

EXPORTED = (
    "mdgemm_opts_init",
    "mdgemm_plan",
    "mdgemm",
    "mdgemm_workspace_bytes",
    "mdgemm_ex",
    "mdgemm_ex_noalloc",
    "mdgemm_workspace_layout",
    "mdgemm_stage_times",
    "mdgemm_status_string",
    "mdgemm_release",
    "mdgemm_exponents",
    "mdgemm_line_spread",
    "mdgemm_split",
    "mdgemm_split_panel",
    "mdgemm_slice_gemm",
    "mdgemm_accumulate",
    "mdgemm_accum_renorm",
    "mdgemm_schedule_info",
    "mdgemm_schedule_export",
    "mdgemm_schedule_workspace_bytes",
    "mdgemm_schedule_levels",
    "mdgemm_qr_dd_workspace_bytes",
    "mdgemm_qr_dd",
    "mdgemm_taylor_dd_workspace_bytes",
    "mdgemm_taylor_dd",
    "mdgemm_probe_mfma_f64",
    "mdgemm_probe_copy",
    "mdgemm_probe_stream",
)


class MdgemmError(RuntimeError):
    def __init__(self, status: int, where: str):
        self.status = status
        super().__init__(f"{where}: {status_string(status)} (status {status})")


class mdgemm_opts(ctypes.Structure):
    _fields_ = [
        ("stream", ctypes.c_void_p),
        ("workspace", ctypes.c_void_p),
        ("workspace_bytes", ctypes.c_size_t),
        ("slices_per_limb", ctypes.c_int),
        ("cutoff", ctypes.c_int),
        ("flags", ctypes.c_uint),
        ("slice_bits", ctypes.c_int),
        ("slices", ctypes.c_int),
        ("range_bits", ctypes.c_int),
    ]


_lib = None
_i64 = ctypes.c_int64
_vp = ctypes.c_void_p


def lib() -> ctypes.CDLL:
    """Load the in-tree ``libmdgemm.so``; raise if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with `python -m paper_2607_06881_amd.build` "
                               "or __graft_entry__.build()")
        L = ctypes.CDLL(LIB_PATH)
        L.mdgemm_opts_init.argtypes = [ctypes.POINTER(mdgemm_opts)]
        L.mdgemm_opts_init.restype = None
        _ip = ctypes.POINTER(ctypes.c_int)
        L.mdgemm_plan.argtypes = [_i64, _i64, _i64, ctypes.c_int, ctypes.POINTER(mdgemm_opts), _ip, _ip, _ip]
        L.mdgemm_plan.restype = ctypes.c_int
        L.mdgemm.argtypes = [_i64, _i64, _i64, ctypes.c_int, _vp, _vp, _vp]
        L.mdgemm.restype = ctypes.c_int
        L.mdgemm_workspace_bytes.argtypes = [_i64, _i64, _i64, ctypes.c_int, ctypes.POINTER(mdgemm_opts)]
        L.mdgemm_workspace_bytes.restype = ctypes.c_size_t
        L.mdgemm_ex.argtypes = [_i64, _i64, _i64, ctypes.c_int, _vp, _vp, _vp, ctypes.POINTER(mdgemm_opts)]
        L.mdgemm_ex.restype = ctypes.c_int
        L.mdgemm_ex_noalloc.argtypes = [_i64, _i64, _i64, ctypes.c_int, _vp, _vp, _vp, ctypes.POINTER(mdgemm_opts)]
        L.mdgemm_ex_noalloc.restype = ctypes.c_int
        L.mdgemm_workspace_layout.argtypes = [_i64, _i64, _i64, ctypes.c_int, ctypes.POINTER(mdgemm_opts),
                                              ctypes.POINTER(ctypes.c_int64), ctypes.c_int]
        L.mdgemm_workspace_layout.restype = ctypes.c_int
        L.mdgemm_stage_times.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_int]
        L.mdgemm_stage_times.restype = ctypes.c_int
        L.mdgemm_status_string.argtypes = [ctypes.c_int]
        L.mdgemm_status_string.restype = ctypes.c_char_p
        L.mdgemm_release.argtypes = []
        L.mdgemm_release.restype = None
        L.mdgemm_exponents.argtypes = [_i64, _i64, ctypes.c_int, _vp, _vp, _vp]
        L.mdgemm_exponents.restype = ctypes.c_int
        L.mdgemm_line_spread.argtypes = [_i64, _i64, ctypes.c_int, _vp, _vp, _vp, _vp]
        L.mdgemm_line_spread.restype = ctypes.c_int
        _c = ctypes.c_int
        L.mdgemm_split.argtypes = [_i64, _i64, _c, _c, _c, _c, _vp, _vp, _vp, _vp]
        L.mdgemm_split.restype = ctypes.c_int
        L.mdgemm_split_panel.argtypes = [_i64, _i64, _c, _c, _c, _c, _vp, _vp, _vp, _vp]
        L.mdgemm_split_panel.restype = ctypes.c_int
        L.mdgemm_slice_gemm.argtypes = [_i64, _i64, _i64, _c, _c, _c, _c, _vp, _vp, _vp, _vp]
        L.mdgemm_slice_gemm.restype = ctypes.c_int
        L.mdgemm_accumulate.argtypes = [_i64, _i64, _c, _c, _vp, _vp, _vp]
        L.mdgemm_accumulate.restype = ctypes.c_int
        L.mdgemm_accum_renorm.argtypes = [_i64, _i64, _c, _c, _c, _vp, _vp, _vp, _vp, _vp]
        L.mdgemm_accum_renorm.restype = ctypes.c_int
        _u = ctypes.c_uint
        L.mdgemm_schedule_info.argtypes = [_i64, _i64, _i64, _c, _c, _c, _u, ctypes.POINTER(ctypes.c_int64), _c]
        L.mdgemm_schedule_info.restype = ctypes.c_int
        L.mdgemm_schedule_export.argtypes = [_i64, _i64, _i64, _c, _c, _c, _u] + [_vp] * 8
        L.mdgemm_schedule_export.restype = ctypes.c_int
        L.mdgemm_schedule_workspace_bytes.argtypes = [_i64, _i64, _i64, _c, _c, _c, _u]
        L.mdgemm_schedule_workspace_bytes.restype = ctypes.c_size_t
        L.mdgemm_schedule_levels.argtypes = [_i64, _i64, _i64, _c, _c, _c, _u, _vp, _vp, _vp, _vp, ctypes.c_size_t,
                                             _vp]
        L.mdgemm_schedule_levels.restype = ctypes.c_int
        L.mdgemm_qr_dd_workspace_bytes.argtypes = [_i64, _i64, ctypes.c_int]
        L.mdgemm_qr_dd_workspace_bytes.restype = ctypes.c_size_t
        L.mdgemm_qr_dd.argtypes = [_i64, _i64, ctypes.c_int, _vp, _vp, _vp, ctypes.c_size_t, _vp]
        L.mdgemm_qr_dd.restype = ctypes.c_int
        L.mdgemm_taylor_dd_workspace_bytes.argtypes = [_i64, _i64, ctypes.c_int]
        L.mdgemm_taylor_dd_workspace_bytes.restype = ctypes.c_size_t
        L.mdgemm_taylor_dd.argtypes = [_i64, _i64, ctypes.c_int, _vp, _vp, _vp, _vp, ctypes.c_size_t, _vp]
        L.mdgemm_taylor_dd.restype = ctypes.c_int
        L.mdgemm_probe_mfma_f64.argtypes = [_i64, _i64, _vp, _vp]
        L.mdgemm_probe_mfma_f64.restype = ctypes.c_int64
        L.mdgemm_probe_copy.argtypes = [_vp, _vp, _i64, _vp]
        L.mdgemm_probe_copy.restype = ctypes.c_int
        L.mdgemm_probe_stream.argtypes = [_vp, ctypes.c_int, _vp, ctypes.c_int, _i64, _vp]
        L.mdgemm_probe_stream.restype = ctypes.c_int
        _lib = L
    return _lib


def status_string(status: int) -> str:
    return lib().mdgemm_status_string(int(status)).decode()


def _check(status: int, where: str) -> None:
    if status != MDGEMM_OK:
        raise MdgemmError(status, where)


def _ptr(t: Optional[torch.Tensor]) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _dev_tensor(t: torch.Tensor, dtype: torch.dtype, name: str) -> None:
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if not t.is_cuda:
        raise ValueError(f"{name} must live on the GPU")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def _stream(stream) -> int:
    if stream is None:
        stream = torch.cuda.current_stream()
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


def make_opts(*, slices_per_limb: int = 0, cutoff: int = MDGEMM_CUTOFF_DEFAULT, flags: int = 0, stream=None,
              workspace: Optional[torch.Tensor] = None, slice_bits: int = 0, slices: int = 0,
              range_bits: int = 0) -> mdgemm_opts:
    o = mdgemm_opts()
    lib().mdgemm_opts_init(ctypes.byref(o))
    o.slices_per_limb = slices_per_limb
    o.cutoff = cutoff
    o.flags = flags
    o.slice_bits = slice_bits
    o.slices = slices
    o.range_bits = range_bits
    o.stream = _stream(stream)
    if workspace is not None:
        o.workspace = workspace.data_ptr()
        o.workspace_bytes = workspace.numel() * workspace.element_size()
    return o


def mdgemm_workspace_bytes(m: int, n: int, k: int, limbs: int, *, slices_per_limb: int = 0,
                           cutoff: int = MDGEMM_CUTOFF_DEFAULT, slice_bits: int = 0, slices: int = 0,
                           range_bits: int = 0, flags: int = 0) -> int:
    o = mdgemm_opts()
    lib().mdgemm_opts_init(ctypes.byref(o))
    o.slices_per_limb = slices_per_limb
    o.cutoff = cutoff
    o.flags = flags
    o.slice_bits = slice_bits
    o.slices = slices
    o.range_bits = range_bits
    return int(lib().mdgemm_workspace_bytes(m, n, k, limbs, ctypes.byref(o)))


def mdgemm_plan(m: int, n: int, k: int, limbs: int, *, slices_per_limb: int = 0,
                cutoff: int = MDGEMM_CUTOFF_DEFAULT, slice_bits: int = 0, slices: int = 0, range_bits: int = 0,
                flags: int = 0):
    """(digit width w, digit count S, cutoff T) that mdgemm_ex uses for these options."""
    o = mdgemm_opts()
    lib().mdgemm_opts_init(ctypes.byref(o))
    o.slices_per_limb = slices_per_limb
    o.cutoff = cutoff
    o.flags = flags
    o.slice_bits = slice_bits
    o.slices = slices
    o.range_bits = range_bits
    w, S, T = ctypes.c_int(), ctypes.c_int(), ctypes.c_int()
    _check(lib().mdgemm_plan(m, n, k, limbs, ctypes.byref(o), ctypes.byref(w), ctypes.byref(S), ctypes.byref(T)),
           "mdgemm_plan")
    return w.value, S.value, T.value


def mdgemm_ex(A: torch.Tensor, B: torch.Tensor, C: Optional[torch.Tensor] = None, *, slices_per_limb: int = 0,
              cutoff: int = MDGEMM_CUTOFF_DEFAULT, flags: int = 0, workspace: Optional[torch.Tensor] = None,
              stream=None, slice_bits: int = 0, slices: int = 0, range_bits: int = 0) -> torch.Tensor:
    """C = A.B for limb-major float64 tensors A [L, m, k] and B [L, k, n] on the GPU.

    The workspace is a torch uint8 tensor (allocated here when not given), so
    device memory comes from PyTorch's allocator."""
    _dev_tensor(A, torch.float64, "A")
    _dev_tensor(B, torch.float64, "B")
    if A.dim() != 3 or B.dim() != 3 or A.shape[0] != B.shape[0] or A.shape[2] != B.shape[1]:
        raise ValueError(f"shapes {tuple(A.shape)} and {tuple(B.shape)} do not form a product [L,m,k].[L,k,n]")
    L, m, k = A.shape
    n = B.shape[2]
    if C is None:
        C = torch.empty((L, m, n), dtype=torch.float64, device=A.device)
    else:
        _dev_tensor(C, torch.float64, "C")
        if tuple(C.shape) != (L, m, n):
            raise ValueError("C has the wrong shape")
    if workspace is None:
        need = mdgemm_workspace_bytes(m, n, k, L, slices_per_limb=slices_per_limb, cutoff=cutoff,
                                      slice_bits=slice_bits, slices=slices, range_bits=range_bits, flags=flags)
        if need == 2**64 - 1:
            _check(MDGEMM_EINVAL, "mdgemm_workspace_bytes")
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=A.device)
    o = make_opts(slices_per_limb=slices_per_limb, cutoff=cutoff, flags=flags, stream=stream, workspace=workspace,
                  slice_bits=slice_bits, slices=slices, range_bits=range_bits)
    _check(lib().mdgemm_ex(m, n, k, L, _ptr(A), _ptr(B), _ptr(C), ctypes.byref(o)), "mdgemm_ex")
    return C


LAYOUT_INFO_KEYS = ("ea", "eb", "da", "db", "planes_off", "panel_bytes", "kp", "mp", "np", "planes",
                    "direct_levels", "total")


def mdgemm_workspace_layout(m: int, n: int, k: int, limbs: int, *, slices_per_limb: int = 0,
                            cutoff: int = MDGEMM_CUTOFF_DEFAULT, slice_bits: int = 0, slices: int = 0,
                            range_bits: int = 0, flags: int = 0) -> dict:
    """Byte offsets and sizes of the parts mdgemm_ex writes into a caller workspace (host only)."""
    o = make_opts(slices_per_limb=slices_per_limb, cutoff=cutoff, flags=flags, slice_bits=slice_bits, slices=slices,
                  range_bits=range_bits, stream=0)
    buf = (ctypes.c_int64 * MDGEMM_LAYOUT_INFO)()
    cnt = lib().mdgemm_workspace_layout(m, n, k, limbs, ctypes.byref(o), buf, MDGEMM_LAYOUT_INFO)
    if cnt < 0:
        _check(cnt, "mdgemm_workspace_layout")
    return {key: int(buf[i]) for i, key in enumerate(LAYOUT_INFO_KEYS[:cnt])}


def workspace_parts(ws: torch.Tensor, m: int, n: int, k: int, limbs: int, **opts) -> dict:
    """Views of a caller workspace after mdgemm_ex: EA [m], EB [n] (int32), the digit
    panels DA [CA, kp, mp], DB [CB, kp, np] (float32 or float64) and the output
    planes G [P, m, n] (float64).  Argument marshalling only (offsets from the library)."""
    lay = mdgemm_workspace_layout(m, n, k, limbs, **opts)
    if ws.numel() < lay["total"]:
        raise ValueError("workspace smaller than the layout")
    pdt = torch.float32 if lay["panel_bytes"] == 4 else torch.float64
    kp, mp, np_ = lay["kp"], lay["mp"], lay["np"]
    ca = (lay["db"] - lay["da"]) // (lay["panel_bytes"] * kp * mp)
    cb = (lay["planes_off"] - lay["db"]) // (lay["panel_bytes"] * kp * np_)

    def view(off, count, dtype, shape):
        size = torch.empty(0, dtype=dtype).element_size()
        return ws[off:off + count * size].view(dtype).view(shape)

    return {
        "layout": lay,
        "EA": view(lay["ea"], m, torch.int32, (m,)),
        "EB": view(lay["eb"], n, torch.int32, (n,)),
        "DA": view(lay["da"], ca * kp * mp, pdt, (ca, kp, mp)),
        "DB": view(lay["db"], cb * kp * np_, pdt, (cb, kp, np_)),
        "G": view(lay["planes_off"], lay["planes"] * m * n, torch.float64, (lay["planes"], m, n)),
    }


def mdgemm_ex_noalloc(A: torch.Tensor, B: torch.Tensor, C: torch.Tensor, *, slices_per_limb: int = 0,
                      cutoff: int = MDGEMM_CUTOFF_DEFAULT, flags: int = 0, stream=None, slice_bits: int = 0,
                      slices: int = 0, range_bits: int = 0) -> torch.Tensor:
    """C = A.B through the allocation-free entry point (the library's fixed device
    scratch instead of a workspace); C must be given."""
    _dev_tensor(A, torch.float64, "A")
    _dev_tensor(B, torch.float64, "B")
    _dev_tensor(C, torch.float64, "C")
    L, m, k = A.shape
    n = B.shape[2]
    if tuple(B.shape) != (L, k, n) or tuple(C.shape) != (L, m, n):
        raise ValueError("shapes do not form a product [L,m,k].[L,k,n] -> [L,m,n]")
    o = make_opts(slices_per_limb=slices_per_limb, cutoff=cutoff, flags=flags, stream=stream, slice_bits=slice_bits,
                  slices=slices, range_bits=range_bits)
    _check(lib().mdgemm_ex_noalloc(m, n, k, L, _ptr(A), _ptr(B), _ptr(C), ctypes.byref(o)), "mdgemm_ex_noalloc")
    return C


def mdgemm(A: torch.Tensor, B: torch.Tensor, C: Optional[torch.Tensor] = None) -> torch.Tensor:
    """C = A.B with the default options through the plain ``mdgemm`` entry point
    (default stream, library-owned workspace)."""
    _dev_tensor(A, torch.float64, "A")
    _dev_tensor(B, torch.float64, "B")
    L, m, k = A.shape
    n = B.shape[2]
    if C is None:
        C = torch.empty((L, m, n), dtype=torch.float64, device=A.device)
    _check(lib().mdgemm(m, n, k, L, _ptr(A), _ptr(B), _ptr(C)), "mdgemm")
    return C


def mdgemm_stage_times() -> list:
    buf = (ctypes.c_float * 4)()
    n = lib().mdgemm_stage_times(buf, 4)
    if n < 0:
        _check(n, "mdgemm_stage_times")
    return [float(buf[i]) for i in range(n)]


def mdgemm_release() -> None:
    lib().mdgemm_release()


def mdgemm_exponents(X0: torch.Tensor, axis: int, E: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """Grid exponents (int32) of every row (axis 0) or column (axis 1) of a [rows, cols] plane."""
    _dev_tensor(X0, torch.float64, "X0")
    rows, cols = X0.shape
    if E is None:
        E = torch.empty(rows if axis == 0 else cols, dtype=torch.int32, device=X0.device)
    _check(lib().mdgemm_exponents(rows, cols, axis, _ptr(X0), _ptr(E), _stream(stream)), "mdgemm_exponents")
    return E


def mdgemm_line_spread(X0: torch.Tensor, axis: int, stream=None):
    """(E, spread) int32 per row (axis 0) or column (axis 1): the grid exponents and
    E minus the smallest exponent of a nonzero entry of the line."""
    _dev_tensor(X0, torch.float64, "X0")
    rows, cols = X0.shape
    lines = rows if axis == 0 else cols
    E = torch.empty(lines, dtype=torch.int32, device=X0.device)
    spread = torch.empty(lines, dtype=torch.int32, device=X0.device)
    _check(lib().mdgemm_line_spread(rows, cols, axis, _ptr(X0), _ptr(E), _ptr(spread), _stream(stream)),
           "mdgemm_line_spread")
    return E, spread


def mdgemm_split(X: torch.Tensor, E: torch.Tensor, slices: int, axis: int, D: Optional[torch.Tensor] = None,
                 stream=None, bits: int = MDGEMM_SLICE_BITS) -> torch.Tensor:
    """Digits [slices, rows, cols] (float64) of `bits` bits of X [L, rows, cols] on the grid exponents E."""
    _dev_tensor(X, torch.float64, "X")
    _dev_tensor(E, torch.int32, "E")
    L, rows, cols = X.shape
    if D is None:
        D = torch.empty((slices, rows, cols), dtype=torch.float64, device=X.device)
    _check(lib().mdgemm_split(rows, cols, L, slices, bits, axis, _ptr(X), _ptr(E), _ptr(D), _stream(stream)),
           "mdgemm_split")
    return D


def mdgemm_split_panel(X: torch.Tensor, E: torch.Tensor, slices: int, axis: int, D: Optional[torch.Tensor] = None,
                       stream=None, bits: int = MDGEMM_SLICE_BITS) -> torch.Tensor:
    """Digits of X [L, rows, cols] as a level-GEMM panel: axis 0 (A):
    [slices, panel_k(cols), panel_mn(rows)] (transposed); axis 1 (B):
    [slices, panel_k(rows), panel_mn(cols)]; zero padding."""
    _dev_tensor(X, torch.float64, "X")
    _dev_tensor(E, torch.int32, "E")
    L, rows, cols = X.shape
    shape = (slices, panel_k(cols), panel_mn(rows)) if axis == 0 else (slices, panel_k(rows), panel_mn(cols))
    if D is None:
        D = torch.empty(shape, dtype=torch.float64, device=X.device)
    _check(lib().mdgemm_split_panel(rows, cols, L, slices, bits, axis, _ptr(X), _ptr(E), _ptr(D),
                                    _stream(stream)), "mdgemm_split_panel")
    return D


def mdgemm_slice_gemm(DAt: torch.Tensor, DBp: torch.Tensor, m: int, n: int, k: int, cutoff: int,
                      per_pair: bool = False, out: Optional[torch.Tensor] = None, stream=None,
                      bits: int = MDGEMM_SLICE_BITS) -> torch.Tensor:
    """Level products [cutoff+1, m, n] (or pair products [S, S, m, n]) of the digit
    panels DAt [S, panel_k(k), panel_mn(m)] and DBp [S, panel_k(k), panel_mn(n)]."""
    _dev_tensor(DAt, torch.float64, "DAt")
    _dev_tensor(DBp, torch.float64, "DBp")
    S = DAt.shape[0]
    if tuple(DAt.shape) != (S, panel_k(k), panel_mn(m)) or tuple(DBp.shape) != (S, panel_k(k), panel_mn(n)):
        raise ValueError("digit panels have the wrong shape")
    if out is None:
        shape = (S, S, m, n) if per_pair else (cutoff + 1, m, n)
        out = torch.zeros(shape, dtype=torch.float64, device=DAt.device)
    _check(lib().mdgemm_slice_gemm(m, n, k, S, bits, cutoff, int(per_pair), _ptr(DAt), _ptr(DBp), _ptr(out),
                                   _stream(stream)), "mdgemm_slice_gemm")
    return out


def mdgemm_accumulate(G: torch.Tensor, Z: Optional[torch.Tensor] = None, stream=None,
                      bits: int = MDGEMM_SLICE_BITS) -> torch.Tensor:
    """Exact sums N = sum_t G_t 2^(w (T - t)), w = bits, as MDGEMM_Z_WORDS int64 words
    [MDGEMM_Z_WORDS, m, n], least significant first."""
    _dev_tensor(G, torch.float64, "G")
    levels, m, n = G.shape
    if Z is None:
        Z = torch.empty((MDGEMM_Z_WORDS, m, n), dtype=torch.int64, device=G.device)
    _check(lib().mdgemm_accumulate(m, n, levels, bits, _ptr(G), _ptr(Z), _stream(stream)), "mdgemm_accumulate")
    return Z


def mdgemm_accum_renorm(G: torch.Tensor, EA: torch.Tensor, EB: torch.Tensor, limbs: int,
                        C: Optional[torch.Tensor] = None, stream=None, bits: int = MDGEMM_SLICE_BITS) -> torch.Tensor:
    """C [limbs, m, n]: exact sum of the levels (weights 2^(-w t), w = bits) rounded greedily
    into limbs, scaled by 2^(EA+EB-2w)."""
    _dev_tensor(G, torch.float64, "G")
    _dev_tensor(EA, torch.int32, "EA")
    _dev_tensor(EB, torch.int32, "EB")
    levels, m, n = G.shape
    if C is None:
        C = torch.empty((limbs, m, n), dtype=torch.float64, device=G.device)
    _check(lib().mdgemm_accum_renorm(m, n, limbs, levels, bits, _ptr(G), _ptr(EA), _ptr(EB), _ptr(C),
                                     _stream(stream)), "mdgemm_accum_renorm")
    return C


SCHEDULE_INFO_KEYS = ("terms", "jobs", "planes", "combos_a", "combos_b", "entries", "max_job_weight", "max_depth",
                      "direct_levels", "max_digits", "panels_f32", "ksplit")


def mdgemm_schedule_info(m: int, n: int, k: int, slices: int, cutoff: int, *, bits: int = MDGEMM_SLICE_BITS,
                         flags: int = 0) -> dict:
    """Sizes of the schedule of the level products of an m x k by k x n product (host only)."""
    buf = (ctypes.c_int64 * MDGEMM_SCHEDULE_INFO)()
    cnt = lib().mdgemm_schedule_info(m, n, k, slices, bits, cutoff, flags, buf, MDGEMM_SCHEDULE_INFO)
    if cnt < 0:
        _check(cnt, "mdgemm_schedule_info")
    return {key: int(buf[i]) for i, key in enumerate(SCHEDULE_INFO_KEYS[:cnt])}


def mdgemm_schedule_export(m: int, n: int, k: int, slices: int, cutoff: int, *, bits: int = MDGEMM_SLICE_BITS,
                           flags: int = 0) -> dict:
    """The schedule's tables as numpy arrays (host only): mask_a/mask_b (uint64 digit
    sets), parents_a/parents_b [C, 2], jobs [J, 4] (first pair, count, plane, k chunk),
    pairs [terms, 2], plane_first [P + 1], entries [E, 2] (level, coefficient)."""
    import numpy as np

    info = mdgemm_schedule_info(m, n, k, slices, cutoff, bits=bits, flags=flags)
    out = {
        "mask_a": np.zeros(info["combos_a"], dtype=np.uint64),
        "parents_a": np.zeros((info["combos_a"], 2), dtype=np.int32),
        "mask_b": np.zeros(info["combos_b"], dtype=np.uint64),
        "parents_b": np.zeros((info["combos_b"], 2), dtype=np.int32),
        "jobs": np.zeros((info["jobs"], 4), dtype=np.int32),
        "pairs": np.zeros((info["terms"], 2), dtype=np.int32),
        "plane_first": np.zeros(info["planes"] + 1, dtype=np.int32),
        "entries": np.zeros((info["entries"], 2), dtype=np.int32),
    }
    order = ("mask_a", "parents_a", "mask_b", "parents_b", "jobs", "pairs", "plane_first", "entries")
    _check(lib().mdgemm_schedule_export(m, n, k, slices, bits, cutoff, flags,
                                        *[out[key].ctypes.data_as(ctypes.c_void_p) for key in order]),
           "mdgemm_schedule_export")
    out["info"] = info
    return out


def mdgemm_schedule_workspace_bytes(m: int, n: int, k: int, slices: int, cutoff: int, *,
                                    bits: int = MDGEMM_SLICE_BITS, flags: int = 0) -> int:
    return int(lib().mdgemm_schedule_workspace_bytes(m, n, k, slices, bits, cutoff, flags))


def mdgemm_schedule_levels(DAt: torch.Tensor, DBp: torch.Tensor, m: int, n: int, k: int, cutoff: int, *,
                           flags: int = 0, bits: int = MDGEMM_SLICE_BITS, out: Optional[torch.Tensor] = None,
                           workspace: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """Levels [cutoff+1, m, n] of the digit panels by the schedule `flags` selects
    (MDGEMM_KARATSUBA or 0); workspace: a torch uint8 tensor, allocated here when
    not given."""
    _dev_tensor(DAt, torch.float64, "DAt")
    _dev_tensor(DBp, torch.float64, "DBp")
    S = DAt.shape[0]
    if tuple(DAt.shape) != (S, panel_k(k), panel_mn(m)) or tuple(DBp.shape) != (S, panel_k(k), panel_mn(n)):
        raise ValueError("digit panels have the wrong shape")
    if out is None:
        out = torch.empty((cutoff + 1, m, n), dtype=torch.float64, device=DAt.device)
    if workspace is None:
        need = mdgemm_schedule_workspace_bytes(m, n, k, S, cutoff, bits=bits, flags=flags)
        if need == 2**64 - 1:
            _check(MDGEMM_EINVAL, "mdgemm_schedule_workspace_bytes")
        workspace = torch.empty(max(need, 1), dtype=torch.uint8, device=DAt.device)
    _check(lib().mdgemm_schedule_levels(m, n, k, S, bits, cutoff, flags, _ptr(DAt), _ptr(DBp), _ptr(out),
                                        _ptr(workspace), workspace.numel(), _stream(stream)),
           "mdgemm_schedule_levels")
    return out


def mdgemm_probe_mfma_f64(sink: torch.Tensor, iters: int, stream=None) -> int:
    """Launch the FP64 MFMA throughput probe with sink.numel() // 256 blocks;
    returns the flops of the launch (time it with events on the same stream)."""
    _dev_tensor(sink, torch.float64, "sink")
    blocks = sink.numel() // 256
    flops = lib().mdgemm_probe_mfma_f64(blocks, iters, _ptr(sink), _stream(stream))
    if flops < 0:
        _check(int(flops), "mdgemm_probe_mfma_f64")
    return int(flops)


def mdgemm_probe_copy(src: torch.Tensor, dst: torch.Tensor, stream=None) -> None:
    """dst = src (float64, same size) through the library's copy probe."""
    _dev_tensor(src, torch.float64, "src")
    _dev_tensor(dst, torch.float64, "dst")
    if src.numel() != dst.numel():
        raise ValueError("src and dst differ in size")
    _check(lib().mdgemm_probe_copy(_ptr(src), _ptr(dst), src.numel(), _stream(stream)), "mdgemm_probe_copy")


def mdgemm_probe_stream(src: torch.Tensor, reads: int, dst: Optional[torch.Tensor], writes: int, count: int,
                        stream=None) -> None:
    """Read `reads` planes of `count` doubles from src and write `writes` planes
    to dst through the library's stream probe."""
    _dev_tensor(src, torch.float64, "src")
    if src.numel() < reads * count:
        raise ValueError("src holds fewer than reads x count doubles")
    if writes > 0:
        _dev_tensor(dst, torch.float64, "dst")
        if dst.numel() < writes * count:
            raise ValueError("dst holds fewer than writes x count doubles")
    _check(lib().mdgemm_probe_stream(_ptr(src), reads, _ptr(dst) if writes > 0 else None, writes, count,
                                     _stream(stream)), "mdgemm_probe_stream")


def mdgemm_qr_dd(A: torch.Tensor, nb: int = 64, workspace: Optional[torch.Tensor] = None, stream=None):
    """Householder QR of a double-double matrix A [2, m, n] (m >= n) in place:
    returns (A, tau) with R on and above the diagonal of A, the Householder
    vectors below it, and tau [2, n]."""
    _dev_tensor(A, torch.float64, "A")
    if A.dim() != 3 or A.shape[0] != 2:
        raise ValueError("A must be a double-double matrix [2, m, n]")
    _, m, n = A.shape
    tau = torch.empty((2, n), dtype=torch.float64, device=A.device)
    if workspace is None:
        need = int(lib().mdgemm_qr_dd_workspace_bytes(m, n, nb))
        if need == 2**64 - 1:
            _check(MDGEMM_EINVAL, "mdgemm_qr_dd_workspace_bytes")
        workspace = torch.empty(need, dtype=torch.uint8, device=A.device)
    _check(lib().mdgemm_qr_dd(m, n, nb, _ptr(A), _ptr(tau), _ptr(workspace), workspace.numel(), _stream(stream)),
           "mdgemm_qr_dd")
    return A, tau


def mdgemm_taylor_dd(A: torch.Tensor, B: torch.Tensor, X: Optional[torch.Tensor] = None,
                     workspace: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """The Taylor coefficients X [d+1, 2, n, r] of the solution of A(t) X(t) = B(t)
    modulo t^(d+1), for the double-double coefficients A [d+1, 2, n, n] and
    B [d+1, 2, n, r] (A_0 nonsingular)."""
    _dev_tensor(A, torch.float64, "A")
    _dev_tensor(B, torch.float64, "B")
    if A.dim() != 4 or A.shape[1] != 2 or A.shape[2] != A.shape[3]:
        raise ValueError("A must hold d + 1 double-double matrices [d + 1, 2, n, n]")
    nd, _, n, _ = A.shape
    if B.dim() != 4 or B.shape[0] != nd or B.shape[1] != 2 or B.shape[2] != n:
        raise ValueError("B must be [d + 1, 2, n, r] with the d and n of A")
    r = B.shape[3]
    if X is None:
        X = torch.empty((nd, 2, n, r), dtype=torch.float64, device=A.device)
    _dev_tensor(X, torch.float64, "X")
    if tuple(X.shape) != (nd, 2, n, r):
        raise ValueError("X must be [d + 1, 2, n, r]")
    if workspace is None:
        need = int(lib().mdgemm_taylor_dd_workspace_bytes(n, r, nd - 1))
        if need == 2**64 - 1:
            _check(MDGEMM_EINVAL, "mdgemm_taylor_dd_workspace_bytes")
        workspace = torch.empty(need, dtype=torch.uint8, device=A.device)
    _check(lib().mdgemm_taylor_dd(n, r, nd - 1, _ptr(A), _ptr(B), _ptr(X), _ptr(workspace), workspace.numel(),
                                  _stream(stream)), "mdgemm_taylor_dd")
    return X
