"""ctypes binding of the C ABI in include/cnn.h (libcnn_mi355x.so).

Argument marshalling only: every step of the convolution runs in the HIP
kernels of the library.  If the library has not been built this module
raises on first use -- there is no fallback implementation.

Tensor arguments are torch tensors on the GPU (device memory and the
current stream are all torch is used for); raw device pointers can be
passed to the ``*_ptr`` variants instead.
"""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libcnn_mi355x.so")

CNN_F32, CNN_BF16, CNN_BF16_OBF16 = 0, 1, 2
DTYPES = {"f32": CNN_F32, "bf16": CNN_BF16, "bf16_obf16": CNN_BF16_OBF16}

(K_AUTO, K_DIRECT, K_IGEMM, K_POINTWISE, K_SMALLC, K_IGEMM_PIPE, K_IGEMM_DMA, K_IGEMM_WIDE,
 K_IGEMM_RAWK) = range(9)
K_ROWS, K_GEMM1, K_SROWS, K_SPLITC, K_AUTO_NO_WORKSPACE = range(10, 15)
KERNEL_NAMES = {K_DIRECT: "direct", K_IGEMM: "igemm", K_POINTWISE: "pointwise", K_SMALLC: "smallc",
                K_IGEMM_PIPE: "igemm_pipe", K_IGEMM_DMA: "igemm_dma", K_IGEMM_WIDE: "igemm_wide",
                K_IGEMM_RAWK: "igemm_rawk", K_ROWS: "rows",
                K_GEMM1: "gemm1", K_SROWS: "srows", K_SPLITC: "splitc"}

STATUS = {0: "CNN_OK", -1: "CNN_E_NULL", -2: "CNN_E_SHAPE", -3: "CNN_E_DTYPE",
          -4: "CNN_E_OVERFLOW", -5: "CNN_E_ALIAS", -6: "CNN_E_UNSUPPORTED",
          -7: "CNN_E_HIP", -8: "CNN_E_PLAN"}

# Every symbol include/cnn.h declares.
EXPORTS = ["cnn_fwd", "cnn_plan", "cnn_plan_candidates", "cnn_variants", "cnn_plan_find",
           "cnn_plan_lookup", "cnn_plan_tiles", "cnn_fwd_plan", "cnn_fwd_plan_ws",
           "cnn_fwd_plan_static", "cnn_eq1_cost",
           "cnn_slab_cost", "cnn_closed_form", "cnn_hbm_bytes", "cnn_device_budget",
           "cnn_strerror", "cnn_last_error", "cnn_abi_version"]

i64 = ctypes.c_int64


class Problem(ctypes.Structure):
    _fields_ = [(n, i64) for n in ("Nb", "Nc", "Nk", "Nw", "Nh", "Nr", "Ns", "sw", "sh")]


class Tiles(ctypes.Structure):
    _fields_ = [(n, i64) for n in ("Tb", "Tk", "Tc", "Tw", "Th")]


class Budget(ctypes.Structure):
    _fields_ = [(n, i64) for n in ("cus", "lds_bytes", "acc_regs", "wg_per_cu")]


class Plan(ctypes.Structure):
    _fields_ = [("prob", Problem), ("dtype", ctypes.c_int32), ("kernel", ctypes.c_int32),
                ("variant", ctypes.c_int32), ("kc", ctypes.c_int32),
                ("tk", i64), ("tp", i64), ("tc", i64), ("grid", i64), ("lds_bytes", i64),
                ("slab_rows", i64), ("ws_bytes", i64), ("eq1_elems", ctypes.c_double * 3),
                ("eq1_bytes", ctypes.c_double), ("compulsory_bytes", ctypes.c_double),
                ("flops", ctypes.c_double), ("mfma_flops", ctypes.c_double),
                ("hbm_bytes", ctypes.c_double), ("model_us", ctypes.c_double)]

    def as_dict(self) -> dict:
        return {"kernel": KERNEL_NAMES.get(self.kernel, str(self.kernel)), "variant": self.variant,
                "tk": self.tk, "tp": self.tp, "tc": self.tc, "grid": self.grid, "kc": self.kc,
                "lds_bytes": self.lds_bytes, "slab_rows": self.slab_rows, "ws_bytes": self.ws_bytes,
                "eq1_elems": list(self.eq1_elems), "eq1_bytes": self.eq1_bytes,
                "compulsory_bytes": self.compulsory_bytes, "flops": self.flops,
                "mfma_flops": self.mfma_flops, "hbm_bytes": self.hbm_bytes,
                "model_us": self.model_us}


class VariantInfo(ctypes.Structure):
    _fields_ = [("kernel", ctypes.c_int32), ("variant", ctypes.c_int32), ("dtype", ctypes.c_int32),
                ("nr", ctypes.c_int32), ("ns", ctypes.c_int32), ("mode", ctypes.c_int32),
                ("tk", i64), ("tp", i64), ("tc", i64)]


class ClosedForm(ctypes.Structure):
    _fields_ = [("M_L", ctypes.c_double), ("Tk", ctypes.c_double), ("Tbhw", ctypes.c_double),
                ("cost", ctypes.c_double), ("row", ctypes.c_int32), ("split_c", ctypes.c_int32)]


class CnnError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{STATUS.get(status, status)}: {message}")
        self.status = status


_lib = None


def lib():
    """The loaded library (raises if it was not built)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"HIP library missing: {LIB_PATH} "
                           "(build it with: python -m paper_2105_13480_amd.build)")
    # The library and torch both need libamdhip64.so.7, and the loader keeps
    # the first one loaded.  Load torch's first: a process whose torch ran
    # on another copy of the HIP runtime finds no GPU.
    import torch  # noqa: F401
    L = ctypes.CDLL(LIB_PATH)
    vp = ctypes.c_void_p
    P, T, B, PL = (ctypes.POINTER(x) for x in (Problem, Tiles, Budget, Plan))
    L.cnn_fwd.argtypes = [vp, vp, vp] + [i64] * 9 + [ctypes.c_int, vp]
    L.cnn_plan.argtypes = [P, ctypes.c_int, B, PL]
    ip = ctypes.POINTER(ctypes.c_int)
    L.cnn_plan_candidates.argtypes = [P, ctypes.c_int, B, PL, ctypes.c_int, ip]
    L.cnn_variants.argtypes = [ctypes.POINTER(VariantInfo), ctypes.c_int, ip]
    L.cnn_plan_find.argtypes = [vp, vp, vp, P, ctypes.c_int, vp, PL, ctypes.POINTER(ctypes.c_double)]
    L.cnn_plan_lookup.argtypes = [P, ctypes.c_int, PL]
    L.cnn_plan_tiles.argtypes = [P, ctypes.c_int, ctypes.c_int, i64, i64, i64, B, PL]
    L.cnn_fwd_plan.argtypes = [vp, vp, vp, P, ctypes.c_int, PL, vp]
    L.cnn_fwd_plan_ws.argtypes = [vp, vp, vp, P, ctypes.c_int, PL, vp, i64, vp]
    L.cnn_fwd_plan_static.argtypes = [vp, vp, vp, P, ctypes.c_int, PL, vp]
    L.cnn_eq1_cost.argtypes = [P, T, ctypes.c_int, ctypes.POINTER(ctypes.c_double),
                               ctypes.POINTER(ctypes.c_double)]
    L.cnn_slab_cost.argtypes = [P, i64, i64, ctypes.POINTER(ctypes.c_double)]
    L.cnn_closed_form.argtypes = [P, ctypes.c_double, ctypes.c_double, ctypes.c_int,
                                  ctypes.POINTER(ClosedForm)]
    L.cnn_hbm_bytes.argtypes = [PL, i64, i64, ctypes.POINTER(ctypes.c_double)]
    L.cnn_device_budget.argtypes = [ctypes.c_int, B]
    L.cnn_strerror.argtypes = [ctypes.c_int]
    L.cnn_strerror.restype = ctypes.c_char_p
    L.cnn_last_error.argtypes = []
    L.cnn_last_error.restype = ctypes.c_char_p
    L.cnn_abi_version.argtypes = []
    for f in ("cnn_fwd", "cnn_plan", "cnn_plan_candidates", "cnn_variants", "cnn_plan_find", "cnn_plan_lookup", "cnn_plan_tiles", "cnn_fwd_plan", "cnn_fwd_plan_ws", "cnn_fwd_plan_static",
              "cnn_eq1_cost", "cnn_slab_cost", "cnn_closed_form", "cnn_hbm_bytes", "cnn_device_budget",
              "cnn_abi_version"):
        getattr(L, f).restype = ctypes.c_int
    _lib = L
    return L


def _check(status: int):
    if status != 0:
        raise CnnError(status, lib().cnn_last_error().decode())


def problem(Nb, Nc, Nk, Nw, Nh, Nr, Ns, sw=1, sh=1) -> Problem:
    return Problem(Nb, Nc, Nk, Nw, Nh, Nr, Ns, sw, sh)


def budget(cus=256, lds_bytes=160 * 1024, acc_regs=128, wg_per_cu=2) -> Budget:
    return Budget(cus, lds_bytes, acc_regs, wg_per_cu)


def device_budget(device: int = 0) -> Budget:
    b = Budget()
    _check(lib().cnn_device_budget(device, ctypes.byref(b)))
    return b


def plan(prob: Problem, dtype: int, bud: Budget | None = None) -> Plan:
    pl = Plan()
    _check(lib().cnn_plan(ctypes.byref(prob), dtype, ctypes.byref(bud) if bud else None,
                          ctypes.byref(pl)))
    return pl


def plan_candidates(prob: Problem, dtype: int, bud: Budget | None = None) -> list:
    """Every candidate plan cnn_plan ranks, with its model fields."""
    n = ctypes.c_int()
    bref = ctypes.byref(bud) if bud else None
    _check(lib().cnn_plan_candidates(ctypes.byref(prob), dtype, bref, None, 0, ctypes.byref(n)))
    arr = (Plan * max(1, n.value))()
    _check(lib().cnn_plan_candidates(ctypes.byref(prob), dtype, bref, arr, n.value,
                                     ctypes.byref(n)))
    return [Plan.from_buffer_copy(arr[i]) for i in range(n.value)]


def variants() -> list:
    """The library's kernel instantiations (cnn_variants)."""
    n = ctypes.c_int()
    _check(lib().cnn_variants(None, 0, ctypes.byref(n)))
    arr = (VariantInfo * max(1, n.value))()
    _check(lib().cnn_variants(arr, n.value, ctypes.byref(n)))
    return [VariantInfo.from_buffer_copy(arr[i]) for i in range(n.value)]


def plan_lookup(prob: Problem, dtype: int) -> Plan:
    """The plan cnn_fwd uses for (prob, dtype) on the current device."""
    pl = Plan()
    _check(lib().cnn_plan_lookup(ctypes.byref(prob), dtype, ctypes.byref(pl)))
    return pl


def plan_tiles(prob: Problem, dtype: int, kernel: int, tk=0, tp=0, tc=0,
               bud: Budget | None = None) -> Plan:
    pl = Plan()
    _check(lib().cnn_plan_tiles(ctypes.byref(prob), dtype, kernel, tk, tp, tc,
                                ctypes.byref(bud) if bud else None, ctypes.byref(pl)))
    return pl


def eq1_cost(prob: Problem, tiles: Tiles, halo: int = 0):
    """(terms[Out, Ker, In], footprint) of Eq. (1); halo 0 = printed, 1 = exact."""
    terms = (ctypes.c_double * 3)()
    fp = ctypes.c_double()
    _check(lib().cnn_eq1_cost(ctypes.byref(prob), ctypes.byref(tiles), halo, terms,
                              ctypes.byref(fp)))
    return tuple(terms), fp.value


def slab_cost(prob: Problem, tk: int, tp: int):
    terms = (ctypes.c_double * 3)()
    _check(lib().cnn_slab_cost(ctypes.byref(prob), tk, tp, terms))
    return tuple(terms)


def closed_form(prob: Problem, P: float, M: float, capacity_mode: int = 0) -> ClosedForm:
    """Table 1 optimum of Eq. (4): capacity_mode 0 = M_L = M (lower bound),
    1 = the relaxed capacity valid for Eq. (3)."""
    out = ClosedForm()
    _check(lib().cnn_closed_form(ctypes.byref(prob), P, M, capacity_mode, ctypes.byref(out)))
    return out


def hbm_bytes(pl: Plan, xcds: int = 8, l2_bytes: int = 4 << 20):
    """(Out, Ker, In) HBM bytes of a plan at the XCD / L2 level (a model)."""
    terms = (ctypes.c_double * 3)()
    _check(lib().cnn_hbm_bytes(ctypes.byref(pl), xcds, l2_bytes, terms))
    return tuple(terms)


# ---- compute entry points ------------------------------------------------

def fwd_ptr(In: int, Ker: int, Out: int, dims, dtype: int, stream: int = 0):
    """cnn_fwd on raw device pointers; dims = (Nb,Nc,Nk,Nw,Nh,Nr,Ns,sw,sh)."""
    _check(lib().cnn_fwd(In, Ker, Out, *dims, dtype, stream))


def fwd_plan_ptr(In: int, Ker: int, Out: int, prob: Problem, dtype: int, pl: Plan,
                 stream: int = 0):
    _check(lib().cnn_fwd_plan(In, Ker, Out, ctypes.byref(prob), dtype, ctypes.byref(pl), stream))


def fwd_plan_ws_ptr(In: int, Ker: int, Out: int, prob: Problem, dtype: int, pl: Plan,
                    ws: int, ws_bytes: int, stream: int = 0):
    _check(lib().cnn_fwd_plan_ws(In, Ker, Out, ctypes.byref(prob), dtype, ctypes.byref(pl),
                                 ws, ws_bytes, stream))


STATIC_SCRATCH_BYTES = 8 << 20


def fwd_plan_static_ptr(In: int, Ker: int, Out: int, prob: Problem, dtype: int, pl: Plan,
                        stream: int = 0):
    _check(lib().cnn_fwd_plan_static(In, Ker, Out, ctypes.byref(prob), dtype, ctypes.byref(pl),
                                     stream))


def _tensor_dims(In, Ker, Out, sw, sh):
    import torch
    for name, t in (("In", In), ("Ker", Ker), ("Out", Out)):
        if not t.is_cuda or not t.is_contiguous():
            raise ValueError(f"{name} must be a contiguous GPU tensor")
        if t.dim() != 4:
            raise ValueError(f"{name} must be 4-d")
    Nb, Nc, Nx, Ny = In.shape
    Nk, Nc2, Nr, Ns = Ker.shape
    if Nc2 != Nc or (Nx - Nr) % sw or (Ny - Ns) % sh or Nx < Nr or Ny < Ns:
        raise ValueError("In extent must be sigma*(N-1)+R and channels must agree")
    Nw, Nh = (Nx - Nr) // sw + 1, (Ny - Ns) // sh + 1
    if tuple(Out.shape) != (Nb, Nk, Nw, Nh):
        raise ValueError(f"Out must have shape {(Nb, Nk, Nw, Nh)}")
    if In.dtype == torch.float32 and Ker.dtype == torch.float32 and Out.dtype == torch.float32:
        dt = CNN_F32
    elif In.dtype == torch.bfloat16 and Ker.dtype == torch.bfloat16:
        if Out.dtype == torch.float32:
            dt = CNN_BF16
        elif Out.dtype == torch.bfloat16:
            dt = CNN_BF16_OBF16
        else:
            raise ValueError("Out must be float32 or bfloat16")
    else:
        raise ValueError("In/Ker must both be float32 or both bfloat16")
    return (Nb, Nc, Nk, Nw, Nh, Nr, Ns, sw, sh), dt


def _stream(stream):
    import torch
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    return getattr(stream, "cuda_stream", stream)


def fwd(In, Ker, Out, sw: int = 1, sh: int = 1, stream=None):
    """Out = conv(In, Ker) on the GPU via cnn_fwd (asynchronous on the
    current torch stream unless ``stream`` is given)."""
    dims, dt = _tensor_dims(In, Ker, Out, sw, sh)
    fwd_ptr(In.data_ptr(), Ker.data_ptr(), Out.data_ptr(), dims, dt, _stream(stream))
    return Out


def plan_find(In, Ker, Out, sw: int = 1, sh: int = 1, stream=None):
    """cnn_plan_find: time every feasible tiling on these buffers, cache and
    return (plan, mean ms) of the fastest.  Synchronises the stream."""
    dims, dt = _tensor_dims(In, Ker, Out, sw, sh)
    pl = Plan()
    ms = ctypes.c_double()
    _check(lib().cnn_plan_find(In.data_ptr(), Ker.data_ptr(), Out.data_ptr(),
                               ctypes.byref(problem(*dims)), dt, _stream(stream),
                               ctypes.byref(pl), ctypes.byref(ms)))
    return pl, ms.value


def fwd_plan(In, Ker, Out, pl: Plan, sw: int = 1, sh: int = 1, stream=None):
    dims, dt = _tensor_dims(In, Ker, Out, sw, sh)
    fwd_plan_ptr(In.data_ptr(), Ker.data_ptr(), Out.data_ptr(), problem(*dims), dt, pl,
                 _stream(stream))
    return Out


def fwd_plan_ws(In, Ker, Out, pl: Plan, workspace, sw: int = 1, sh: int = 1, stream=None):
    """cnn_fwd_plan_ws with a caller-owned workspace tensor (any dtype, on the GPU)."""
    dims, dt = _tensor_dims(In, Ker, Out, sw, sh)
    ws_ptr = workspace.data_ptr() if workspace is not None else 0
    ws_bytes = workspace.numel() * workspace.element_size() if workspace is not None else 0
    fwd_plan_ws_ptr(In.data_ptr(), Ker.data_ptr(), Out.data_ptr(), problem(*dims), dt, pl,
                    ws_ptr, ws_bytes, _stream(stream))
    return Out


def fwd_plan_static(In, Ker, Out, pl: Plan, sw: int = 1, sh: int = 1, stream=None):
    """cnn_fwd_plan_static: the plan's workspace is the library's static
    device scratch (no allocation; calls that overlap on one GPU race)."""
    dims, dt = _tensor_dims(In, Ker, Out, sw, sh)
    fwd_plan_static_ptr(In.data_ptr(), Ker.data_ptr(), Out.data_ptr(), problem(*dims), dt, pl,
                        _stream(stream))
    return Out
