"""ctypes binding of libspconv.so (include/spconv.h).

Argument marshalling only: torch supplies device memory (``torch.empty``) and the
current HIP stream; every step of the layer runs in the library's HIP kernels.
There is no fallback: if the library is not built, importing the functions
raises.
"""
from __future__ import annotations

import ctypes
import os

import torch

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libspconv.so")

SPCONV_OK, SPCONV_EINVAL, SPCONV_ERANGE, SPCONV_EDUP, SPCONV_ENOSPC, SPCONV_EHIP, SPCONV_EUNSUPPORTED = (
    0, -1, -2, -3, -4, -5, -6)
SPCONV_SUBM, SPCONV_DOWN, SPCONV_UP = 0, 1, 2
SPCONV_F32, SPCONV_F16, SPCONV_BF16 = 0, 1, 2
GROUP_RAGGED, GROUP_SORTED, GROUP_MAPORDER = 0, 1, 2
GATHER_BUFFER, GATHER_FUSED = 1, 2
MODES = {"subm": SPCONV_SUBM, "down": SPCONV_DOWN, "up": SPCONV_UP}
DTYPES = {torch.float32: SPCONV_F32, torch.float16: SPCONV_F16, torch.bfloat16: SPCONV_BF16}
TORCH_DTYPES = {"f32": torch.float32, "f16": torch.float16, "bf16": torch.bfloat16}

EXPORTED = [
    "spconv_map_workspace_bytes", "spconv_build_map", "spconv_map_transpose", "spconv_map_n_in",
    "spconv_map_n_out", "spconv_map_kvol", "spconv_map_out_coords", "spconv_map_counts",
    "spconv_map_pairs", "spconv_map_copy_pairs", "spconv_map_copy_out_coords", "spconv_free_map",
    "spconv_forward_workspace_bytes", "spconv_forward", "spconv_forward_ex", "spconv_forward_noalloc",
    "spconv_concat_rows",
    "spconv_forward_plan", "spconv_profile_enable", "spconv_profile_phase_count",
    "spconv_profile_phase_name", "spconv_profile_read", "spconv_last_error",
]


class SpconvError(RuntimeError):
    def __init__(self, status: int, where: str, msg: str):
        super().__init__(f"{where}: status {status}: {msg}")
        self.status = status


class Options(ctypes.Structure):
    _fields_ = [("B", ctypes.c_int), ("Cq", ctypes.c_int), ("t_gather", ctypes.c_int),
                ("t_scatter", ctypes.c_int), ("grouping", ctypes.c_int), ("partial_dtype", ctypes.c_int),
                ("launch_cost_rows", ctypes.c_int), ("presorted", ctypes.c_int), ("search", ctypes.c_int),
                ("gather", ctypes.c_int), ("wg", ctypes.c_int), ("gemm_tile_rows", ctypes.c_int),
                ("centre", ctypes.c_int), ("count_group", ctypes.c_int), ("reserved", ctypes.c_int * 2)]

    @classmethod
    def make(cls, **kw) -> "Options":
        o = cls()
        for k, v in kw.items():
            if k == "grouping" and v is not None:
                v = int(v) + 1
            setattr(o, k, int(v or 0))
        return o


class PlanInfo(ctypes.Structure):
    _fields_ = [("rows_real", ctypes.c_int64), ("rows_padded", ctypes.c_int64),
                ("n_gemm_launches", ctypes.c_int), ("t_gather", ctypes.c_int), ("t_scatter", ctypes.c_int),
                ("grouping", ctypes.c_int), ("gather", ctypes.c_int), ("centre", ctypes.c_int)]


_lib = None


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run __graft_entry__.build() (no CPU fallback exists)")
    L = ctypes.CDLL(LIB_PATH)
    vp, i64, i32, c_int, sz = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_int, ctypes.c_size_t
    optp = ctypes.POINTER(Options)
    L.spconv_map_workspace_bytes.argtypes = [i64, i64, c_int, c_int, optp]
    L.spconv_map_workspace_bytes.restype = sz
    L.spconv_build_map.argtypes = [vp, i64, vp, i64, c_int, c_int, c_int, c_int, optp, vp, sz, vp,
                                   ctypes.POINTER(vp)]
    L.spconv_build_map.restype = c_int
    L.spconv_map_transpose.argtypes = [vp, ctypes.POINTER(vp)]
    L.spconv_map_transpose.restype = c_int
    for n in ("spconv_map_n_in", "spconv_map_n_out"):
        getattr(L, n).argtypes = [vp]
        getattr(L, n).restype = i64
    L.spconv_map_kvol.argtypes = [vp]
    L.spconv_map_kvol.restype = c_int
    L.spconv_map_out_coords.argtypes = [vp]
    L.spconv_map_out_coords.restype = vp
    L.spconv_map_counts.argtypes = [vp, ctypes.POINTER(i64)]
    L.spconv_map_counts.restype = c_int
    L.spconv_map_pairs.argtypes = [vp, c_int, ctypes.POINTER(vp), ctypes.POINTER(vp), ctypes.POINTER(i64)]
    L.spconv_map_pairs.restype = c_int
    L.spconv_map_copy_pairs.argtypes = [vp, vp, vp, vp]
    L.spconv_map_copy_pairs.restype = c_int
    L.spconv_map_copy_out_coords.argtypes = [vp, vp, vp]
    L.spconv_map_copy_out_coords.restype = c_int
    L.spconv_free_map.argtypes = [vp]
    L.spconv_free_map.restype = None
    L.spconv_forward_workspace_bytes.argtypes = [vp, c_int, c_int, c_int, optp]
    L.spconv_forward_workspace_bytes.restype = sz
    L.spconv_forward.argtypes = [vp, vp, vp, vp, c_int, c_int, c_int, optp, vp, sz, vp]
    L.spconv_forward.restype = c_int
    L.spconv_forward_ex.argtypes = [vp, vp, vp, vp, c_int, c_int, c_int, vp, c_int, optp, vp, sz, vp]
    L.spconv_forward_ex.restype = c_int
    L.spconv_forward_noalloc.argtypes = [vp, vp, vp, vp, c_int, c_int, c_int, vp, c_int, optp, vp]
    L.spconv_forward_noalloc.restype = c_int
    L.spconv_concat_rows.argtypes = [vp, c_int, vp, c_int, vp, i64, c_int, vp]
    L.spconv_concat_rows.restype = c_int
    L.spconv_forward_plan.argtypes = [vp, c_int, c_int, c_int, optp, ctypes.POINTER(PlanInfo)]
    L.spconv_forward_plan.restype = c_int
    L.spconv_profile_enable.argtypes = [ctypes.c_uint64]
    L.spconv_profile_enable.restype = c_int
    L.spconv_profile_phase_count.argtypes = []
    L.spconv_profile_phase_count.restype = c_int
    L.spconv_profile_phase_name.argtypes = [c_int]
    L.spconv_profile_phase_name.restype = ctypes.c_char_p
    L.spconv_profile_read.argtypes = [ctypes.POINTER(ctypes.c_double), ctypes.POINTER(i64), c_int, c_int]
    L.spconv_profile_read.restype = c_int
    L.spconv_last_error.argtypes = []
    L.spconv_last_error.restype = ctypes.c_char_p
    _ = i32
    _lib = L
    return L


def _check(st: int, where: str):
    if st != SPCONV_OK:
        raise SpconvError(st, where, lib().spconv_last_error().decode(errors="replace"))


def _ptr(t: torch.Tensor | None):
    return ctypes.c_void_p(t.data_ptr()) if t is not None and t.numel() > 0 else ctypes.c_void_p(0)


def _stream(stream=None):
    if stream is None:
        # the current stream's raw handle, without building a Stream object
        return ctypes.c_void_p(torch._C._cuda_getCurrentRawStream(torch.cuda.current_device()))
    return ctypes.c_void_p(stream.cuda_stream)


def _opt(opt: Options | None):
    return ctypes.byref(opt) if opt is not None else None


# ----------------------------------------------------------------------------
# Same names as the C-ABI (marshalling only)
# ----------------------------------------------------------------------------

def spconv_map_workspace_bytes(n_in: int, n_out: int, K: int, mode: int, opt: Options | None = None) -> int:
    return int(lib().spconv_map_workspace_bytes(n_in, n_out, K, mode, _opt(opt)))


def spconv_build_map(in_coords: torch.Tensor, out_coords: torch.Tensor | None, K: int, stride: int,
                     tensor_stride: int, mode: int, opt: Options | None, workspace: torch.Tensor,
                     stream=None) -> ctypes.c_void_p:
    h = ctypes.c_void_p()
    n_out = 0 if out_coords is None else out_coords.shape[0]
    st = lib().spconv_build_map(_ptr(in_coords), in_coords.shape[0], _ptr(out_coords), n_out, K, stride,
                                tensor_stride, mode, _opt(opt), _ptr(workspace), workspace.numel(),
                                _stream(stream), ctypes.byref(h))
    _check(st, "spconv_build_map")
    return h


def spconv_map_transpose(down) -> ctypes.c_void_p:
    h = ctypes.c_void_p()
    _check(lib().spconv_map_transpose(down, ctypes.byref(h)), "spconv_map_transpose")
    return h


def spconv_map_counts(m) -> list[int]:
    k3 = lib().spconv_map_kvol(m)
    arr = (ctypes.c_int64 * k3)()
    _check(lib().spconv_map_counts(m, arr), "spconv_map_counts")
    return list(arr)


def spconv_map_pairs(m, k: int):
    a, b, n = ctypes.c_void_p(), ctypes.c_void_p(), ctypes.c_int64()
    _check(lib().spconv_map_pairs(m, k, ctypes.byref(a), ctypes.byref(b), ctypes.byref(n)), "spconv_map_pairs")
    return a.value, b.value, n.value


def spconv_free_map(m) -> None:
    lib().spconv_free_map(m)


def spconv_forward_workspace_bytes(m, c_in: int, c_out: int, dtype: int, opt: Options | None = None) -> int:
    return int(lib().spconv_forward_workspace_bytes(m, c_in, c_out, dtype, _opt(opt)))


def spconv_forward(m, x: torch.Tensor, w: torch.Tensor, y: torch.Tensor, c_in: int, c_out: int, dtype: int,
                   opt: Options | None, workspace: torch.Tensor, stream=None) -> None:
    st = lib().spconv_forward(m, _ptr(x), _ptr(w), _ptr(y), c_in, c_out, dtype, _opt(opt), _ptr(workspace),
                              workspace.numel(), _stream(stream))
    _check(st, "spconv_forward")


def spconv_forward_ex(m, x: torch.Tensor, w: torch.Tensor, y: torch.Tensor, c_in: int, c_out: int, dtype: int,
                      residual: torch.Tensor | None, relu: bool, opt: Options | None, workspace: torch.Tensor,
                      stream=None) -> None:
    st = lib().spconv_forward_ex(m, _ptr(x), _ptr(w), _ptr(y), c_in, c_out, dtype, _ptr(residual), 1 if relu else 0,
                                 _opt(opt), _ptr(workspace), workspace.numel(), _stream(stream))
    _check(st, "spconv_forward_ex")


def spconv_forward_noalloc(m, x: torch.Tensor, w: torch.Tensor, y: torch.Tensor, c_in: int, c_out: int,
                           dtype: int, residual: torch.Tensor | None = None, relu: bool = False,
                           opt: Options | None = None, stream=None) -> None:
    st = lib().spconv_forward_noalloc(m, _ptr(x), _ptr(w), _ptr(y), c_in, c_out, dtype, _ptr(residual),
                                      1 if relu else 0, _opt(opt), _stream(stream))
    _check(st, "spconv_forward_noalloc")


def spconv_concat_rows(a: torch.Tensor, b: torch.Tensor, out: torch.Tensor | None = None, stream=None) -> torch.Tensor:
    if a.shape[0] != b.shape[0] or a.dtype != b.dtype:
        raise ValueError("row counts / dtypes differ")
    if out is None:
        out = torch.empty((a.shape[0], a.shape[1] + b.shape[1]), dtype=a.dtype, device=a.device)
    st = lib().spconv_concat_rows(_ptr(a), a.shape[1], _ptr(b), b.shape[1], _ptr(out), a.shape[0], DTYPES[a.dtype],
                                  _stream(stream))
    _check(st, "spconv_concat_rows")
    return out


def spconv_forward_plan(m, c_in: int, c_out: int, dtype: int, opt: Options | None = None) -> PlanInfo:
    info = PlanInfo()
    _check(lib().spconv_forward_plan(m, c_in, c_out, dtype, _opt(opt), ctypes.byref(info)), "spconv_forward_plan")
    return info


def profile_ids() -> dict:
    """name -> id of every timed phase (ids < 16) and kernel (names start with 'k_')."""
    n = lib().spconv_profile_phase_count()
    out = {}
    for i in range(n):
        name = lib().spconv_profile_phase_name(i).decode()
        if name:
            out[name] = i
    return out


PHASES_ALL = (1 << 16) - 1


def spconv_profile_enable(mask) -> None:
    """mask: an int bit mask of ids, True (all phases and kernels) or False (off)."""
    if mask is True:
        mask = (1 << 64) - 1
    elif mask is False or mask is None:
        mask = 0
    lib().spconv_profile_enable(ctypes.c_uint64(int(mask)))


def spconv_profile_read(reset: bool = True) -> dict:
    """name -> (summed ms, number of timed intervals) for every id that has a name."""
    n = lib().spconv_profile_phase_count()
    ms = (ctypes.c_double * n)()
    cnt = (ctypes.c_int64 * n)()
    _check(lib().spconv_profile_read(ms, cnt, n, 1 if reset else 0), "spconv_profile_read")
    out = {}
    for i in range(n):
        name = lib().spconv_profile_phase_name(i).decode()
        if name:
            out[name] = (ms[i], cnt[i])
    return out


# ----------------------------------------------------------------------------
# Owners for handle + workspace lifetimes
# ----------------------------------------------------------------------------

def _device_bytes(n: int, device) -> torch.Tensor:
    return torch.empty(max(int(n), 1), dtype=torch.uint8, device=device)


class KernelMap:
    """A built kernel map: the library handle plus the device workspace it lives in."""

    def __init__(self, handle, workspace, keep=(), parent=None):
        self.handle = handle
        self.workspace = workspace
        self._keep = keep        # caller coordinate tensors the map points into
        self._parent = parent    # transposed maps borrow their parent's arrays

    @classmethod
    def build(cls, in_coords: torch.Tensor, K: int, stride: int = 1, tensor_stride: int = 1, mode="subm",
              out_coords: torch.Tensor | None = None, opt: Options | None = None, stream=None) -> "KernelMap":
        m = MODES[mode] if isinstance(mode, str) else int(mode)
        n_out = out_coords.shape[0] if (m == SPCONV_UP and out_coords is not None) else 0
        ws = _device_bytes(spconv_map_workspace_bytes(in_coords.shape[0], n_out, K, m, opt), in_coords.device)
        h = spconv_build_map(in_coords, out_coords if m == SPCONV_UP else None, K, stride, tensor_stride, m, opt,
                             ws, stream)
        return cls(h, ws, keep=(in_coords, out_coords))

    def transpose(self) -> "KernelMap":
        return KernelMap(spconv_map_transpose(self.handle), None, parent=self)

    @property
    def n_in(self) -> int:
        return int(lib().spconv_map_n_in(self.handle))

    @property
    def n_out(self) -> int:
        return int(lib().spconv_map_n_out(self.handle))

    @property
    def kvol(self) -> int:
        return int(lib().spconv_map_kvol(self.handle))

    def counts(self) -> list[int]:
        return spconv_map_counts(self.handle)

    @property
    def device(self):
        return self.workspace.device if self.workspace is not None else self._parent.device

    def out_coords(self) -> torch.Tensor:
        """Copy of the output coordinates (device int32 [n_out][4])."""
        out = torch.empty((self.n_out, 4), dtype=torch.int32, device=self.device)
        _check(lib().spconv_map_copy_out_coords(self.handle, _ptr(out), _stream()), "spconv_map_copy_out_coords")
        return out

    def all_pairs(self) -> tuple[torch.Tensor, torch.Tensor, list[int]]:
        """Copies of all pairs, offset-major, plus |M_k| (device int32)."""
        cnt = self.counts()
        m = sum(cnt)
        pin = torch.empty(m, dtype=torch.int32, device=self.device)
        pout = torch.empty(m, dtype=torch.int32, device=self.device)
        _check(lib().spconv_map_copy_pairs(self.handle, _ptr(pin), _ptr(pout), _stream()), "spconv_map_copy_pairs")
        return pin, pout, cnt

    def plan(self, c_in: int, c_out: int, dtype: torch.dtype, opt: Options | None = None) -> PlanInfo:
        return spconv_forward_plan(self.handle, c_in, c_out, DTYPES[dtype], opt)

    def __del__(self):
        h = getattr(self, "handle", None)
        if h is not None and h.value:
            try:
                spconv_free_map(h)
            except Exception:
                pass
            self.handle = None


class Forward:
    """Reusable GMaS workspace for one (map, c_in, c_out, dtype, options)."""

    def __init__(self, kmap: KernelMap, c_in: int, c_out: int, dtype: torch.dtype, opt: Options | None = None):
        self.kmap, self.c_in, self.c_out, self.dtype, self.opt = kmap, c_in, c_out, dtype, opt
        dev = kmap.device
        self.plan = spconv_forward_plan(kmap.handle, c_in, c_out, DTYPES[dtype], opt)  # raises on bad args
        n = spconv_forward_workspace_bytes(kmap.handle, c_in, c_out, DTYPES[dtype], opt)
        self.workspace = _device_bytes(n, dev)
        self.device = dev

    def __call__(self, x: torch.Tensor, w: torch.Tensor, y: torch.Tensor | None = None, stream=None,
                 residual: torch.Tensor | None = None, relu: bool = False) -> torch.Tensor:
        if y is None:
            y = torch.empty((self.kmap.n_out, self.c_out), dtype=self.dtype, device=self.device)
        checks = [(x, (self.kmap.n_in, self.c_in)), (w, (self.kmap.kvol, self.c_in, self.c_out)),
                  (y, (self.kmap.n_out, self.c_out))]
        if residual is not None:
            checks.append((residual, (self.kmap.n_out, self.c_out)))
        for t, shape in checks:
            if tuple(t.shape) != shape or t.dtype != self.dtype or not t.is_contiguous():
                raise ValueError(f"expected contiguous {self.dtype} {shape}, got {t.dtype} {tuple(t.shape)}")
        if residual is None and not relu:
            spconv_forward(self.kmap.handle, x, w, y, self.c_in, self.c_out, DTYPES[self.dtype], self.opt,
                           self.workspace, stream)
        else:
            spconv_forward_ex(self.kmap.handle, x, w, y, self.c_in, self.c_out, DTYPES[self.dtype], residual, relu,
                              self.opt, self.workspace, stream)
        return y


def conv(in_coords: torch.Tensor, x: torch.Tensor, w: torch.Tensor, K: int, stride: int = 1,
         tensor_stride: int = 1, mode="subm", out_coords: torch.Tensor | None = None,
         opt: Options | None = None):
    """One sparse-conv layer through the library: returns (kernel map, y)."""
    km = KernelMap.build(in_coords, K, stride, tensor_stride, mode, out_coords, opt)
    f = Forward(km, x.shape[1], w.shape[2], x.dtype, opt)
    return km, f(x, w)
