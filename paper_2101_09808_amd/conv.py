"""Python binding of the C ABI in ``include/conv_fwd.h`` (ctypes).

Argument marshalling only: every step of the computation runs in the HIP
library ``libconvfwd.so``.  PyTorch provides device memory and the current
stream.  There is no fallback: if the library is missing, or a tensor is not
on the GPU, the call raises.
"""
import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libconvfwd.so")

CONV_OK, CONV_EINVAL, CONV_ENULL, CONV_ERANGE, CONV_ENOPLAN, CONV_EHIP, CONV_ESCRATCH = 0, -1, -2, -3, -4, -5, -6
CONV_NOALLOC_SCRATCH_BYTES = 64 * 1024 * 1024
CONV_DTYPE_F32, CONV_DTYPE_BF16 = 0, 1
LEVELS = ("reg", "lds", "l2", "hbm")
ITER_CODE = {"n": 0, "k": 1, "c": 2, "r": 3, "s": 4, "h": 5, "w": 6}

_i32, _i64, _dbl, _vp = ctypes.c_int, ctypes.c_int64, ctypes.c_double, ctypes.c_void_p


class ConvPlan(ctypes.Structure):
    """Mirror of ``conv_plan_t``."""
    _fields_ = [
        ("dtype", _i32), ("variant", _i32), ("tile_k", _i32), ("tile_rows", _i32),
        ("tile_cols", _i32), ("tile_c", _i32), ("wave_k", _i32), ("wave_px", _i32),
        ("waves_k", _i32), ("waves_px", _i32), ("grid_order", _i32), ("split_c", _i32),
        ("reserved", _i32), ("lds_bytes", _i32), ("num_wg", _i64), ("class_lvl", _i32 * 4), ("pred_bytes", _dbl * 4),
        ("pred_us", _dbl * 4), ("pred_mfma_us", _dbl), ("pred_total_us", _dbl), ("rank_us", _dbl),
        ("paper_bytes", _dbl * 4),
    ]

    def to_dict(self):
        d = {f: getattr(self, f) for f, _ in self._fields_[:15] if f != "reserved"}
        d["class_lvl"] = dict(zip(LEVELS, list(self.class_lvl)))
        d["pred_bytes"] = dict(zip(LEVELS, list(self.pred_bytes)))
        d["pred_us"] = dict(zip(LEVELS, list(self.pred_us)))
        d["pred_mfma_us"] = self.pred_mfma_us
        d["pred_total_us"] = self.pred_total_us
        d["rank_us"] = self.rank_us
        d["paper_bytes"] = dict(zip(LEVELS, list(self.paper_bytes)))
        return d

    @classmethod
    def from_dict(cls, d):
        p = cls()
        for f, _ in cls._fields_[:15]:
            if f in d:
                setattr(p, f, d[f])
        return p


class ConvError(RuntimeError):
    def __init__(self, status, what):
        self.status = status
        super().__init__(f"{what}: {strerror(status)} (status {status})")


_lib = None


def lib():
    """The loaded HIP library (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing; build it with `python -m paper_2101_09808_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        shape7 = [_i32] * 7
        L.conv_fwd.argtypes = shape7 + [_vp, _vp, _vp, _vp]
        L.conv_fwd.restype = _i32
        L.conv_fwd_bf16.argtypes = shape7 + [_vp, _vp, _vp, _vp]
        L.conv_fwd_bf16.restype = _i32
        L.conv_fwd_plan.argtypes = shape7 + [_i32, ctypes.POINTER(ConvPlan)]
        L.conv_fwd_plan.restype = _i32
        L.conv_fwd_with_plan.argtypes = shape7 + [_vp, _vp, _vp, ctypes.POINTER(ConvPlan), _vp]
        L.conv_fwd_with_plan.restype = _i32
        L.conv_fwd_bf16_out_plan.argtypes = shape7 + [ctypes.POINTER(ConvPlan)]
        L.conv_fwd_bf16_out_plan.restype = _i32
        L.conv_fwd_score_plan.argtypes = shape7 + [ctypes.POINTER(ConvPlan)]
        L.conv_fwd_score_plan.restype = _i32
        L.conv_fwd_candidates.argtypes = shape7 + [_i32, ctypes.POINTER(ConvPlan), _i32]
        L.conv_fwd_candidates.restype = _i32
        L.conv_fwd_tune.argtypes = shape7 + [_i32, _vp, _vp, _vp, _i32, _i32, _vp, ctypes.POINTER(ConvPlan),
                                             ctypes.POINTER(ctypes.c_float)]
        L.conv_fwd_tune.restype = _i32
        L.conv_fwd_bf16_out.argtypes = shape7 + [_vp, _vp, _vp, _vp]
        L.conv_fwd_bf16_out.restype = _i32
        L.conv_fwd_ex.argtypes = shape7 + [_i32] * 5 + [_vp, _vp, _vp, _vp]
        L.conv_fwd_ex.restype = _i32
        L.conv_fwd_ex_noalloc.argtypes = shape7 + [_i32] * 5 + [_vp, _vp, _vp, _vp]
        L.conv_fwd_ex_noalloc.restype = _i32
        L.conv_fwd_ex_inner_shape.argtypes = shape7 + [_i32] * 4 + [ctypes.POINTER(_i32)]
        L.conv_fwd_ex_inner_shape.restype = _i32
        L.conv_model_volume.argtypes = [ctypes.POINTER(_i32), ctypes.POINTER(_i64),
                                        ctypes.POINTER(_i64), _i32, ctypes.POINTER(_dbl)]
        L.conv_model_volume.restype = _i32
        L.conv_fwd_geometry.argtypes = shape7 + [ctypes.POINTER(ConvPlan), ctypes.POINTER(_i32), _i32]
        L.conv_fwd_geometry.restype = _i32
        L.conv_fwd_ex_geometry.argtypes = shape7 + [_i32] * 4 + [ctypes.POINTER(ConvPlan), ctypes.POINTER(_i32),
                                                                 _i32]
        L.conv_fwd_ex_geometry.restype = _i32
        L.conv_fwd_ex_plan.argtypes = shape7 + [_i32] * 5 + [ctypes.POINTER(ConvPlan), ctypes.POINTER(_i32)]
        L.conv_fwd_ex_plan.restype = _i32
        L.conv_fwd_release_workspaces.argtypes = [_vp]
        L.conv_fwd_release_workspaces.restype = _i32
        L.conv_fwd_strerror.argtypes = [_i32]
        L.conv_fwd_strerror.restype = ctypes.c_char_p
        _lib = L
    return _lib


def release_workspaces(stream=None):
    """Free the workspaces the library keeps for `stream` (default: the
    current stream) on the current device, in stream order."""
    st = lib().conv_fwd_release_workspaces(_stream_ptr(stream))
    if st != CONV_OK:
        raise ConvError(st, "conv_fwd_release_workspaces")


def strerror(status):
    return lib().conv_fwd_strerror(int(status)).decode()


def _stream_ptr(stream):
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _check_inputs(In, Ker, dtype):
    if not (isinstance(In, torch.Tensor) and isinstance(Ker, torch.Tensor)):
        raise TypeError("In and Ker must be torch tensors")
    if not (In.is_cuda and Ker.is_cuda):
        raise ValueError("In and Ker must be GPU tensors (the library has no CPU path)")
    if In.dtype != dtype or Ker.dtype != dtype:
        raise TypeError(f"expected {dtype} tensors, got {In.dtype} and {Ker.dtype}")
    if In.dim() != 4 or Ker.dim() != 4:
        raise ValueError("In must be [N,C,H,W] and Ker [K,C,R,S]")
    if not (In.is_contiguous() and Ker.is_contiguous()):
        raise ValueError("In and Ker must be contiguous (NCHW / KCRS)")
    N, C, H, W = In.shape
    K, C2, R, S = Ker.shape
    if C2 != C:
        raise ValueError(f"channel mismatch: In has {C}, Ker has {C2}")
    return N, C, K, H, W, R, S


def _out_for(In, shape, out):
    N, C, K, H, W, R, S = shape
    oshape = (N, K, H - R + 1, W - S + 1)
    if out is None:
        return torch.empty(oshape, dtype=torch.float32, device=In.device)
    if out.shape != oshape or out.dtype != torch.float32 or not out.is_contiguous() or out.device != In.device:
        raise ValueError(f"out must be a contiguous float32 {oshape} tensor on {In.device}")
    return out


def conv_fwd(In, Ker, out=None, stream=None):
    """Eq. (1) for fp32 In [N,C,H,W] and Ker [K,C,R,S]; returns fp32 Out [N,K,P,Q]."""
    shape = _check_inputs(In, Ker, torch.float32)
    out = _out_for(In, shape, out)
    st = lib().conv_fwd(*shape, In.data_ptr(), Ker.data_ptr(), out.data_ptr(), _stream_ptr(stream))
    if st != CONV_OK:
        raise ConvError(st, "conv_fwd")
    return out


def conv_fwd_ptr(N, C, K, H, W, R, S, in_ptr, ker_ptr, out_ptr, stream_ptr, bf16=False):
    """Raw-pointer call for tight loops (device addresses as ints, stream as
    an int hipStream_t); returns the status code instead of raising."""
    f = lib().conv_fwd_bf16 if bf16 else lib().conv_fwd
    return f(N, C, K, H, W, R, S, in_ptr, ker_ptr, out_ptr, stream_ptr)


def conv_fwd_bf16(In, Ker, out=None, stream=None):
    """Eq. (1) for bf16 In and Ker, fp32 accumulation and fp32 Out."""
    shape = _check_inputs(In, Ker, torch.bfloat16)
    out = _out_for(In, shape, out)
    st = lib().conv_fwd_bf16(*shape, In.data_ptr(), Ker.data_ptr(), out.data_ptr(), _stream_ptr(stream))
    if st != CONV_OK:
        raise ConvError(st, "conv_fwd_bf16")
    return out


def conv_fwd_bf16_out(In, Ker, out=None, stream=None):
    """Eq. (1) for bf16 In and Ker with fp32 accumulation, Out rounded to
    bf16 (nearest even); returns a bf16 [N,K,P,Q] tensor."""
    shape = _check_inputs(In, Ker, torch.bfloat16)
    N, C, K, H, W, R, S = shape
    oshape = (N, K, H - R + 1, W - S + 1)
    if out is None:
        out = torch.empty(oshape, dtype=torch.bfloat16, device=In.device)
    elif out.shape != oshape or out.dtype != torch.bfloat16 or not out.is_contiguous():
        raise ValueError(f"out must be a contiguous bfloat16 {oshape} tensor")
    st = lib().conv_fwd_bf16_out(*shape, In.data_ptr(), Ker.data_ptr(), out.data_ptr(), _stream_ptr(stream))
    if st != CONV_OK:
        raise ConvError(st, "conv_fwd_bf16_out")
    return out


def conv_fwd_with_plan(In, Ker, plan, out=None, stream=None):
    """Eq. (1) with an explicit tile plan (a ConvPlan or its dict)."""
    if isinstance(plan, dict):
        plan = ConvPlan.from_dict(plan)
    dtype = torch.bfloat16 if plan.dtype == CONV_DTYPE_BF16 else torch.float32
    shape = _check_inputs(In, Ker, dtype)
    out = _out_for(In, shape, out)
    st = lib().conv_fwd_with_plan(*shape, In.data_ptr(), Ker.data_ptr(), out.data_ptr(),
                                  ctypes.byref(plan), _stream_ptr(stream))
    if st != CONV_OK:
        raise ConvError(st, "conv_fwd_with_plan")
    return out


def _pair(x):
    return (int(x), int(x)) if isinstance(x, int) else (int(x[0]), int(x[1]))


def conv_fwd_ex(In, Ker, stride=1, pad=0, out=None, stream=None):
    """Strided, zero-padded convolution (fp32 or bf16 In/Ker, fp32 Out
    [N,K,P,Q] with P = (H + 2 ph - R) // sh + 1, Q likewise)."""
    return _conv_fwd_ex("conv_fwd_ex", In, Ker, stride, pad, out, stream)


def conv_fwd_ex_noalloc(In, Ker, stride=1, pad=0, out=None, stream=None):
    """conv_fwd_ex through the allocation-free entry point: the library's
    workspaces come from its static per-GPU scratch array (out=None still
    lets torch allocate Out; pass `out` to allocate nothing)."""
    return _conv_fwd_ex("conv_fwd_ex_noalloc", In, Ker, stride, pad, out, stream)


def _conv_fwd_ex(fn, In, Ker, stride, pad, out, stream):
    sh, sw = _pair(stride)
    ph, pw = _pair(pad)
    bf16 = In.dtype == torch.bfloat16
    N, C, K, H, W, R, S = _check_inputs(In, Ker, torch.bfloat16 if bf16 else torch.float32)
    inner = conv_fwd_ex_inner_shape(N, C, K, H, W, R, S, (sh, sw), (ph, pw))
    P, Q = inner[7], inner[8]
    if out is None:
        out = torch.empty((N, K, P, Q), dtype=torch.float32, device=In.device)
    elif out.shape != (N, K, P, Q) or out.dtype != torch.float32 or not out.is_contiguous():
        raise ValueError(f"out must be a contiguous float32 {(N, K, P, Q)} tensor")
    st = getattr(lib(), fn)(N, C, K, H, W, R, S, sh, sw, ph, pw, CONV_DTYPE_BF16 if bf16 else CONV_DTYPE_F32,
                            In.data_ptr(), Ker.data_ptr(), out.data_ptr(), _stream_ptr(stream))
    if st != CONV_OK:
        raise ConvError(st, fn)
    return out


def conv_fwd_ex_inner_shape(N, C, K, H, W, R, S, stride=1, pad=0):
    """The stride-1 problem conv_fwd_ex runs: (N, C', K, H', W', R', S', P, Q)."""
    sh, sw = _pair(stride)
    ph, pw = _pair(pad)
    buf = (_i32 * 9)()
    st = lib().conv_fwd_ex_inner_shape(N, C, K, H, W, R, S, sh, sw, ph, pw, buf)
    if st != CONV_OK:
        raise ConvError(st, "conv_fwd_ex_inner_shape")
    return tuple(buf)


CONV_TUNE_MAX = 64


def conv_fwd_tune(In, Ker, top_n=5, reps=3, out=None, stream=None):
    """Time the model's `top_n` best plans on these tensors and keep the
    fastest as the shape's cached plan (Sec. 10, MOpt-5).  In/Ker are fp32
    or bf16.  Blocks until the timed launches have run.  Returns (out, the
    chosen plan as a dict, median launch time in us of each timed plan in the
    model's order -- the first candidates that suit the tensors' alignment)."""
    dtype = CONV_DTYPE_BF16 if In.dtype == torch.bfloat16 else CONV_DTYPE_F32
    shape = _check_inputs(In, Ker, torch.bfloat16 if dtype == CONV_DTYPE_BF16 else torch.float32)
    out = _out_for(In, shape, out)
    plan = ConvPlan()
    times = (ctypes.c_float * max(1, min(int(top_n), CONV_TUNE_MAX)))()
    n = lib().conv_fwd_tune(*shape, dtype, In.data_ptr(), Ker.data_ptr(), out.data_ptr(), int(top_n),
                            int(reps), _stream_ptr(stream), ctypes.byref(plan), times)
    if n < 0:
        raise ConvError(n, "conv_fwd_tune")
    return out, plan.to_dict(), [float(times[i]) for i in range(n)]


def conv_fwd_plan(N, C, K, H, W, R, S, dtype=CONV_DTYPE_F32):
    """The selector's plan for a shape (host only) as a dict."""
    p = ConvPlan()
    st = lib().conv_fwd_plan(N, C, K, H, W, R, S, dtype, ctypes.byref(p))
    if st != CONV_OK:
        raise ConvError(st, "conv_fwd_plan")
    return p.to_dict()


def conv_fwd_bf16_out_plan(N, C, K, H, W, R, S):
    """The plan conv_fwd_bf16_out runs for a shape with a 16-byte aligned
    Out (host only), as a dict."""
    p = ConvPlan()
    st = lib().conv_fwd_bf16_out_plan(N, C, K, H, W, R, S, ctypes.byref(p))
    if st != CONV_OK:
        raise ConvError(st, "conv_fwd_bf16_out_plan")
    return p.to_dict()


def conv_fwd_score_plan(N, C, K, H, W, R, S, plan):
    """The selector's score of a plan's tile fields (host only), as a dict;
    raises ConvError(CONV_EINVAL) for a plan the kernels cannot run."""
    p = ConvPlan.from_dict(plan) if isinstance(plan, dict) else plan
    st = lib().conv_fwd_score_plan(N, C, K, H, W, R, S, ctypes.byref(p))
    if st != CONV_OK:
        raise ConvError(st, "conv_fwd_score_plan")
    return p.to_dict()


def conv_fwd_candidates(N, C, K, H, W, R, S, dtype=CONV_DTYPE_F32, cap=4096):
    """All candidate plans the selector scores for a shape, best first."""
    buf = (ConvPlan * cap)()
    n = lib().conv_fwd_candidates(N, C, K, H, W, R, S, dtype, buf, cap)
    if n < 0:
        raise ConvError(n, "conv_fwd_candidates")
    return [buf[i].to_dict() for i in range(min(n, cap))]


def conv_model_volume(perm, N, T, out_factor=2):
    """The paper's single-level volumes (In, Ker, Out) for a permutation of
    'nkcrshw' (outermost first) and dicts of extents / tile sizes."""
    order = [ITER_CODE[x] for x in perm]
    keys = sorted(ITER_CODE, key=ITER_CODE.get)
    Na = (_i64 * 7)(*[int(N[k]) for k in keys])
    Ta = (_i64 * 7)(*[int(T[k]) for k in keys])
    dv = (_dbl * 3)()
    st = lib().conv_model_volume((_i32 * 7)(*order), Na, Ta, out_factor, dv)
    if st != CONV_OK:
        raise ConvError(st, "conv_model_volume")
    return {"In": dv[0], "Ker": dv[1], "Out": dv[2]}


GEOM_FIELDS = (
    "N", "C", "K", "H", "W", "R", "S", "P", "Q",
    "tr", "tw", "tiles_rows", "tiles_cols", "tiles_k",
    "in_rows", "in_wp", "in_cstride", "ker_rstride",
    "nwk", "nwp", "order", "num_tiles",
    "lds_in_elems", "lds_ker_elems", "ni_in", "ni_ker", "nchunks",
    "wk", "wp", "tc", "rc", "sc", "max_ni", "max_nk", "ker_vec", "threads", "lds_bytes",
    "family", "in_vec", "stages", "stage_elems", "in_region", "in_bytes", "ker_bytes", "grid",
    "phase_skip", "reserved1", "reserved2", "split", "cps", "mfma32", "nwc",
    "nph", "na", "nb", "sh", "sw", "ph", "pw", "C0", "H0", "W0", "Wi",
) + tuple(f"dv_{d}_{x}" for d in ("in_cstride", "in_wp", "H", "ker_rstride", "tw", "P", "nph", "nb", "Wi",
                                  "tiles_k", "tiles_cols", "tiles_rows") for x in ("m", "s"))


def conv_fwd_geometry(N, C, K, H, W, R, S, plan):
    """The launch geometry a plan resolves to (host only), as a dict."""
    if isinstance(plan, dict):
        plan = ConvPlan.from_dict(plan)
    buf = (_i32 * len(GEOM_FIELDS))()
    st = lib().conv_fwd_geometry(N, C, K, H, W, R, S, ctypes.byref(plan), buf, len(GEOM_FIELDS))
    if st < 0:
        raise ConvError(st, "conv_fwd_geometry")
    return _geom_dict(buf)


def _geom_dict(buf):
    d = dict(zip(GEOM_FIELDS, list(buf)[:len(GEOM_FIELDS)]))
    for k in d:
        if k.startswith("dv_") and k.endswith("_m"):
            d[k] &= 0xFFFFFFFF  # multipliers are uint32 bit patterns
    return d


def conv_fwd_ex_plan(N, C, K, H, W, R, S, stride=1, pad=0, dtype=CONV_DTYPE_F32):
    """(plan, direct): the plan conv_fwd_ex runs for this layer (a plan of its
    inner stride-1 problem, host only), and whether its kernel reads In
    through the phase mapping instead of a phase-split copy."""
    sh, sw = _pair(stride)
    ph, pw = _pair(pad)
    p = ConvPlan()
    d = _i32(0)
    st = lib().conv_fwd_ex_plan(N, C, K, H, W, R, S, sh, sw, ph, pw, dtype, ctypes.byref(p), ctypes.byref(d))
    if st != CONV_OK:
        raise ConvError(st, "conv_fwd_ex_plan")
    return p.to_dict(), bool(d.value)


def conv_fwd_ex_geometry(N, C, K, H, W, R, S, stride, pad, plan):
    """The launch geometry conv_fwd_ex uses for `plan` (a plan of its inner
    stride-1 problem), with the direct phase-addressing fields (host only)."""
    if isinstance(plan, dict):
        plan = ConvPlan.from_dict(plan)
    sh, sw = _pair(stride)
    ph, pw = _pair(pad)
    buf = (_i32 * len(GEOM_FIELDS))()
    st = lib().conv_fwd_ex_geometry(N, C, K, H, W, R, S, sh, sw, ph, pw, ctypes.byref(plan), buf,
                                    len(GEOM_FIELDS))
    if st < 0:
        raise ConvError(st, "conv_fwd_ex_geometry")
    return _geom_dict(buf)
