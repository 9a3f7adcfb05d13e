"""Python binding of libattn.so: the C ABI names, argument marshalling only.

Every computation runs in the HIP library; this module converts torch
tensors and Python values into pointers and integers and raises AttnError on
a non-zero status.  Loading the library touches no GPU, so descriptor,
derivation and argument-check entry points work on a host without one.
If the library has not been built, load() raises; there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os

HERE = os.path.dirname(os.path.abspath(__file__))
# ATTN_LIB names another build of this library (the host-sanitizer build of the tests).
LIB_PATH = os.environ.get("ATTN_LIB") or os.path.join(HERE, "libattn.so")

ATTN_BF16 = 0
ATTN_F16 = 1
ATTN_F32 = 2  # attn_gemm only
ATTN_MAX_L = 1 << 24

STATUS = {
    0: "ATTN_OK", -1: "ATTN_E_NULLPTR", -2: "ATTN_E_SHAPE", -3: "ATTN_E_UNSUPPORTED_D",
    -4: "ATTN_E_DTYPE", -5: "ATTN_E_ALIGN", -6: "ATTN_E_INFEASIBLE", -7: "ATTN_E_NO_INSTANCE",
    -8: "ATTN_E_HIP", -9: "ATTN_E_WORKSPACE", -10: "ATTN_E_SCALE", -11: "ATTN_E_ARG",
    -12: "ATTN_E_DEVICE", -13: "ATTN_E_SCRATCH",
}
CODE = {v: k for k, v in STATUS.items()}

# ATTN_NOALLOC_SCRATCH_BYTES of the header: the static split workspace of attn_fwd_noalloc.
NOALLOC_SCRATCH_BYTES = 32 << 20

# Every function the header declares; the CPU tests check each is exported.
EXPORTS = (
    "attn_hw_desc_preset", "attn_hw_desc_query", "attn_atom_preset", "attn_fwd_op",
    "attn_vgpr_estimate", "attn_tile_derive", "attn_fwd_plan", "attn_fwd", "attn_fwd_workspace_bytes",
    "attn_fwd_partial", "attn_fwd_merge", "attn_fwd_unfused",
    "attn_unfused_workspace_bytes", "attn_mfma_probe", "attn_strerror",
    "attn_softmax_derive", "attn_softmax", "attn_gemm_derive", "attn_gemm", "attn_fwd_noalloc",
)

c_int, c_int32, c_int64, c_float, c_double, c_char, c_size_t, c_void_p, c_char_p = (
    ctypes.c_int, ctypes.c_int32, ctypes.c_int64, ctypes.c_float, ctypes.c_double,
    ctypes.c_char, ctypes.c_size_t, ctypes.c_void_p, ctypes.c_char_p)


class _Struct(ctypes.Structure):
    def as_dict(self):
        out = {}
        for name, _ in self._fields_:
            v = getattr(self, name)
            out[name] = v.decode() if isinstance(v, bytes) else v
        return out


class HwDesc(_Struct):
    _fields_ = [("lds_bytes", c_int64), ("vgpr_per_thread", c_int32), ("wavefront_size", c_int32),
                ("num_cus", c_int32), ("simds_per_cu", c_int32), ("lds_bytes_per_clk", c_int32),
                ("mfma_flops_per_clk_cu", c_int32), ("hbm_tbps", c_double), ("peak_tflops", c_double),
                ("clock_ghz", c_double), ("name", c_char * 32)]


class Atom(_Struct):
    _fields_ = [("m", c_int32), ("n", c_int32), ("k", c_int32), ("in_bytes", c_int32),
                ("acc_bytes", c_int32)]


class Op(_Struct):
    _fields_ = [("B", c_int32), ("H", c_int32), ("L", c_int32), ("d", c_int32),
                ("elem_bytes", c_int32), ("causal", c_int32), ("kv_lds_num", c_int32),
                ("kv_lds_den", c_int32), ("kv_tiles", c_int32), ("stage_tiles", c_int32), ("score_tiles", c_int32),
                ("p_tiles", c_int32), ("stat_regs", c_int32), ("operand_frags", c_int32),
                ("waves_per_wg", c_int32), ("waves_per_simd", c_int32), ("vgpr_fixed", c_int32),
                ("max_split", c_int32), ("wg_fixed_steps", c_int32)]


class TileReport(_Struct):
    _fields_ = [("feasible", c_int32), ("t_kv", c_int32), ("t_q_wave", c_int32),
                ("n_waves", c_int32), ("tile_q", c_int32), ("n_split", c_int32),
                ("tiles_per_split", c_int32), ("grid", c_int64), ("vgpr_est", c_int32), ("vgpr_budget", c_int32),
                ("lds_used", c_int64), ("lds_budget", c_int64), ("wg_per_cu", c_double),
                ("low_occupancy", c_int32), ("lds_bw_ok", c_int32), ("binding", c_char * 16),
                ("launch_grid", c_int64)]


class SoftmaxReport(_Struct):
    _fields_ = [("feasible", c_int32), ("tile_elems", c_int32), ("resident_tiles", c_int32),
                ("split", c_int32), ("waves_per_wg", c_int32), ("rows_per_wg", c_int32),
                ("seg", c_int64), ("grid", c_int64), ("passes", c_int32), ("vgpr_est", c_int32),
                ("vgpr_budget", c_int32), ("wg_per_cu", c_double), ("hbm_bytes", c_int64),
                ("binding", c_char * 16)]


class GemmReport(_Struct):
    _fields_ = [("feasible", c_int32), ("t_m", c_int32), ("t_n", c_int32), ("t_k", c_int32),
                ("warp_m", c_int32), ("warp_n", c_int32), ("stages", c_int32), ("waves_per_wg", c_int32),
                ("grid", c_int64), ("vgpr_est", c_int32), ("vgpr_budget", c_int32), ("lds_used", c_int64),
                ("lds_budget", c_int64), ("wg_per_cu", c_double), ("binding", c_char * 16)]


class AttnError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__(f"{STATUS.get(status, status)}: {msg}")
        self.status = status


_lib = None


def load():
    """Load libattn.so (no GPU access).  Raises if it has not been built."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run __graft_entry__.build()")
    # The library needs libamdhip64.so.7, and torch ships its own copy of that
    # HIP runtime under another file name.  Loaded after torch's, the library
    # binds to torch's copy and one runtime serves both (torch's streams and
    # device pointers are valid in its calls); loaded first, it would bring in
    # the system copy and torch a second one.
    try:
        import torch  # noqa: F401
    except ImportError:
        pass
    lib = ctypes.CDLL(LIB_PATH)
    P = ctypes.POINTER
    sig = {
        "attn_hw_desc_preset": (c_int, [c_char_p, P(HwDesc)]),
        "attn_hw_desc_query": (c_int, [c_int, P(HwDesc)]),
        "attn_atom_preset": (c_int, [c_char_p, P(Atom)]),
        "attn_fwd_op": (c_int, [c_int, c_int, c_int, c_int, c_int, c_int, P(Op)]),
        "attn_vgpr_estimate": (c_int, [P(HwDesc), P(Atom), P(Op), c_int, c_int, c_int, P(c_int32)]),
        "attn_tile_derive": (c_int, [P(HwDesc), P(Atom), P(Op), P(TileReport)]),
        "attn_fwd_plan": (c_int, [P(HwDesc), c_int, c_int, c_int, c_int, c_int, c_int, P(TileReport)]),
        "attn_fwd": (c_int, [c_void_p, c_void_p, c_void_p, c_void_p, c_int, c_int, c_int, c_int,
                             c_float, c_int, c_int, c_void_p]),
        "attn_fwd_noalloc": (c_int, [c_void_p, c_void_p, c_void_p, c_void_p, c_int, c_int, c_int, c_int,
                                     c_float, c_int, c_int, c_void_p]),
        "attn_fwd_workspace_bytes": (c_int, [c_int, c_int, c_int, c_int, c_int, c_int, P(c_size_t)]),
        "attn_fwd_partial": (c_int, [c_void_p, c_void_p, c_void_p, c_void_p, c_int, c_int, c_int, c_int,
                                     c_float, c_int, c_int, c_void_p, c_size_t, c_void_p]),
        "attn_fwd_merge": (c_int, [c_void_p, c_size_t, c_void_p, c_int, c_int, c_int, c_int, c_float, c_int,
                                   c_int, c_void_p]),
        "attn_fwd_unfused": (c_int, [c_void_p, c_void_p, c_void_p, c_void_p, c_int, c_int, c_int,
                                     c_int, c_float, c_int, c_int, c_void_p, c_size_t, c_void_p]),
        "attn_unfused_workspace_bytes": (c_size_t, [c_int, c_int, c_int, c_int]),
        "attn_mfma_probe": (c_int, [c_int, c_void_p, c_void_p, c_void_p, c_void_p]),
        "attn_softmax_derive": (c_int, [P(HwDesc), c_int64, c_int64, c_int, P(SoftmaxReport)]),
        "attn_softmax": (c_int, [c_void_p, c_void_p, c_int64, c_int64, c_int, c_int, c_void_p]),
        "attn_gemm_derive": (c_int, [P(HwDesc), P(Atom), c_int64, c_int64, c_int64, P(GemmReport)]),
        "attn_gemm": (c_int, [c_void_p, c_void_p, c_void_p, c_int64, c_int64, c_int64, c_int, c_void_p]),
        "attn_strerror": (c_char_p, [c_int]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def _check(rc):
    if rc != 0:
        raise AttnError(rc, load().attn_strerror(rc).decode())
    return rc


# ------------------------------------------------------------ host-side calls

def attn_hw_desc_preset(name: str) -> HwDesc:
    d = HwDesc()
    _check(load().attn_hw_desc_preset(name.encode(), ctypes.byref(d)))
    return d


def attn_hw_desc_query(device: int = 0) -> HwDesc:
    d = HwDesc()
    _check(load().attn_hw_desc_query(device, ctypes.byref(d)))
    return d


def attn_atom_preset(name: str) -> Atom:
    a = Atom()
    _check(load().attn_atom_preset(name.encode(), ctypes.byref(a)))
    return a


def attn_fwd_op(B, H, L, d, causal, dtype) -> Op:
    o = Op()
    _check(load().attn_fwd_op(B, H, L, d, int(causal), dtype, ctypes.byref(o)))
    return o


def attn_vgpr_estimate(hw: HwDesc, atom: Atom, op: Op, t_q_wave, t_kv, n_waves) -> int:
    out = c_int32()
    _check(load().attn_vgpr_estimate(ctypes.byref(hw), ctypes.byref(atom), ctypes.byref(op),
                                     t_q_wave, t_kv, n_waves, ctypes.byref(out)))
    return out.value


def attn_tile_derive(hw: HwDesc, atom: Atom, op: Op):
    """Returns (status, TileReport); ATTN_E_INFEASIBLE is a result, not an exception."""
    r = TileReport()
    rc = load().attn_tile_derive(ctypes.byref(hw), ctypes.byref(atom), ctypes.byref(op), ctypes.byref(r))
    if rc not in (0, CODE["ATTN_E_INFEASIBLE"]):
        _check(rc)
    return rc, r


def attn_fwd_plan(B, H, L, d, causal, dtype, hw: HwDesc | None = None) -> TileReport:
    r = TileReport()
    _check(load().attn_fwd_plan(ctypes.byref(hw) if hw is not None else None, B, H, L, d,
                                int(causal), dtype, ctypes.byref(r)))
    return r


def attn_unfused_workspace_bytes(B, H, L, dtype) -> int:
    return load().attn_unfused_workspace_bytes(B, H, L, dtype)


def attn_strerror(status: int) -> str:
    return load().attn_strerror(status).decode()


# ------------------------------------------------------------ device calls

# torch glue, looked up once: the dtype codes and torch's current-stream
# getter (the raw handle as an integer, without building a Stream object).
_DTYPES = None
_RAW_STREAM = None


def _torch_glue():
    global _DTYPES, _RAW_STREAM
    import torch
    _RAW_STREAM = getattr(torch._C, "_cuda_getCurrentRawStream", None)
    _DTYPES = {torch.bfloat16: ATTN_BF16, torch.float16: ATTN_F16}
    return _DTYPES


def dtype_code(t) -> int:
    code = (_DTYPES or _torch_glue()).get(t.dtype)
    if code is None:
        raise AttnError(CODE["ATTN_E_DTYPE"], f"unsupported tensor dtype {t.dtype}")
    return code


def _stream_ptr(t, stream):
    """The HIP stream handle: `stream`'s, else torch's current stream on t's device."""
    if stream is None:
        if _DTYPES is None:
            _torch_glue()
        if _RAW_STREAM is not None:
            return _RAW_STREAM(t.get_device())
        import torch
        stream = torch.cuda.current_stream(t.device)
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


def _dev_ptr(t):
    if not t.is_cuda:
        raise AttnError(CODE["ATTN_E_ARG"], "tensor must be on the GPU")
    if not t.is_contiguous():
        raise AttnError(CODE["ATTN_E_ARG"], "tensor must be contiguous [B, H, L, d]")
    return t.data_ptr()


def _same(q, k, v, o):
    shape, dt = q.shape, q.dtype
    for t in (k, v, o):
        if t.shape != shape or t.dtype != dt:
            raise AttnError(CODE["ATTN_E_SHAPE"], "q, k, v, o must share shape and dtype")


def attn_fwd(q, k, v, o, scale: float, causal: bool, stream=None):
    """Enqueue the fused forward on `stream` (default: torch's current stream)."""
    B, H, L, d = q.shape
    _same(q, k, v, o)
    _check(load().attn_fwd(_dev_ptr(q), _dev_ptr(k), _dev_ptr(v), _dev_ptr(o), B, H, L, d,
                           float(scale), int(causal), dtype_code(q), _stream_ptr(q, stream)))


def attn_fwd_noalloc(q, k, v, o, scale: float, causal: bool, stream=None):
    """attn_fwd with the split workspace in the library's static per-GPU array
    (no allocation; calls that overlap on one GPU race on it)."""
    B, H, L, d = q.shape
    _same(q, k, v, o)
    _check(load().attn_fwd_noalloc(_dev_ptr(q), _dev_ptr(k), _dev_ptr(v), _dev_ptr(o), B, H, L, d,
                                   float(scale), int(causal), dtype_code(q), _stream_ptr(q, stream)))


def attn_fwd_workspace_bytes(B, H, L, d, causal, dtype) -> int:
    out = c_size_t()
    _check(load().attn_fwd_workspace_bytes(B, H, L, d, int(causal), dtype, ctypes.byref(out)))
    return out.value


def _ws(workspace):
    if workspace is None:
        return None, 0
    return _dev_ptr(workspace), workspace.numel() * workspace.element_size()


def attn_fwd_partial(q, k, v, o, scale: float, causal: bool, workspace=None, stream=None):
    B, H, L, d = q.shape
    _same(q, k, v, o)
    ws, nb = _ws(workspace)
    _check(load().attn_fwd_partial(_dev_ptr(q), _dev_ptr(k), _dev_ptr(v), _dev_ptr(o), B, H, L, d, float(scale),
                                   int(causal), dtype_code(q), ws, nb, _stream_ptr(q, stream)))


def attn_fwd_merge(workspace, o, scale: float, causal: bool, stream=None):
    B, H, L, d = o.shape
    ws, nb = _ws(workspace)
    _check(load().attn_fwd_merge(ws, nb, _dev_ptr(o), B, H, L, d, float(scale), int(causal), dtype_code(o),
                                 _stream_ptr(o, stream)))


def attn_fwd_unfused(q, k, v, o, scale: float, causal: bool, workspace, stream=None):
    B, H, L, d = q.shape
    _same(q, k, v, o)
    nbytes = workspace.numel() * workspace.element_size()
    _check(load().attn_fwd_unfused(_dev_ptr(q), _dev_ptr(k), _dev_ptr(v), _dev_ptr(o), B, H, L, d,
                                   float(scale), int(causal), dtype_code(q), _dev_ptr(workspace),
                                   nbytes, _stream_ptr(q, stream)))


def attn_mfma_probe(atom: int, a, b, c, stream=None):
    """a: [16, 32], b: [32, 16] (bf16 or f16 device tensors), c: [16, 16] float32 device tensor."""
    _check(load().attn_mfma_probe(atom, _dev_ptr(a), _dev_ptr(b), _dev_ptr(c), _stream_ptr(a, stream)))


def attn_softmax_derive(hw: HwDesc, rows: int, n: int, elem_bytes: int = 2) -> SoftmaxReport:
    r = SoftmaxReport()
    _check(load().attn_softmax_derive(ctypes.byref(hw), rows, n, elem_bytes, ctypes.byref(r)))
    return r


def attn_softmax(x, y, causal: bool = False, stream=None):
    """y = softmax(x) along the last dimension (x, y contiguous, same shape and dtype; y may be x)."""
    if tuple(y.shape) != tuple(x.shape) or y.dtype != x.dtype:
        raise AttnError(CODE["ATTN_E_SHAPE"], "x and y must share shape and dtype")
    n = x.shape[-1]
    rows = x.numel() // n if n else 0
    _check(load().attn_softmax(_dev_ptr(x), _dev_ptr(y), rows, n, int(causal), dtype_code(x),
                               _stream_ptr(x, stream)))


def attn_gemm_derive(hw: HwDesc, atom: Atom, M: int, N: int, K: int) -> GemmReport:
    r = GemmReport()
    _check(load().attn_gemm_derive(ctypes.byref(hw), ctypes.byref(atom), M, N, K, ctypes.byref(r)))
    return r


def attn_gemm(a, b, c, stream=None):
    """c = a @ b: a [M, K] and b [K, N] contiguous device tensors of one dtype
    (bf16, f16 or float32), c [M, N] contiguous float32."""
    import torch
    if a.dim() != 2 or b.dim() != 2 or c.dim() != 2:
        raise AttnError(CODE["ATTN_E_SHAPE"], "a, b and c must be matrices")
    M, K = a.shape
    if b.shape[0] != K or tuple(c.shape) != (M, b.shape[1]):
        raise AttnError(CODE["ATTN_E_SHAPE"], f"shapes {tuple(a.shape)} @ {tuple(b.shape)} -> {tuple(c.shape)}")
    if b.dtype != a.dtype:
        raise AttnError(CODE["ATTN_E_DTYPE"], "a and b must share a dtype")
    if c.dtype != torch.float32:
        raise AttnError(CODE["ATTN_E_DTYPE"], "c must be float32")
    code = ATTN_F32 if a.dtype == torch.float32 else dtype_code(a)
    _check(load().attn_gemm(_dev_ptr(a), _dev_ptr(b), _dev_ptr(c), M, b.shape[1], K, code, _stream_ptr(a, stream)))
