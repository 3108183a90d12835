"""Python binding of libtilemix.so (TileMix routed prefill attention for MI355X / gfx950).

Argument marshalling only: every step of the attention path runs in the HIP kernels of
libtilemix.so.  PyTorch provides device memory and streams.  The functions carry the names
of the C entry points declared in include/tilemix.h.  Importing this module does not load
the library; the first call does, and raises if it has not been built
(``python paper_2608_17336_amd/build.py`` or ``__graft_entry__.build()``).
"""

from __future__ import annotations

import ctypes
import math
import os
from dataclasses import dataclass

__all__ = [
    "TilemixError",
    "Params",
    "library_path",
    "load_library",
    "tilemix_route_words_per_row",
    "tilemix_workspace_size",
    "tilemix_prefill",
    "tilemix_fused_workspace_size",
    "tilemix_prefill_fused",
    "tilemix_prefill_noalloc",
    "tilemix_prepare",
    "tilemix_attend",
    "tilemix_quantize",
    "tilemix_debug_qk_int32",
    "Template",
    "TEMPLATE_KINDS",
    "tilemix_auto_group_size",
    "tilemix_route_template",
    "tilemix_route_template_varlen",
    "tilemix_route_coverage",
    "tilemix_fit_template",
    "tilemix_varlen_workspace_size",
    "tilemix_prefill_varlen",
    "tilemix_varlen_fused_workspace_size",
    "tilemix_prefill_varlen_fused",
    "tilemix_debug_prefill",
    "tilemix_quantize_kv",
    "tilemix_decode_workspace_size",
    "tilemix_decode",
    "tilemix_decode_varlen",
    "EXPORTED_SYMBOLS",
]

EXPORTED_SYMBOLS = (
    "tilemix_route_words_per_row",
    "tilemix_workspace_size",
    "tilemix_prefill",
    "tilemix_fused_workspace_size",
    "tilemix_prefill_fused",
    "tilemix_prefill_noalloc",
    "tilemix_prepare",
    "tilemix_attend",
    "tilemix_quantize",
    "tilemix_debug_qk_int32",
    "tilemix_auto_group_size",
    "tilemix_route_template",
    "tilemix_route_template_varlen",
    "tilemix_route_coverage",
    "tilemix_fit_template",
    "tilemix_varlen_workspace_size",
    "tilemix_prefill_varlen",
    "tilemix_varlen_fused_workspace_size",
    "tilemix_prefill_varlen_fused",
    "tilemix_debug_prefill",
    "tilemix_quantize_kv",
    "tilemix_decode_workspace_size",
    "tilemix_decode",
    "tilemix_decode_varlen",
    "tilemix_status_string",
    "tilemix_last_error",
)

_HERE = os.path.dirname(os.path.abspath(__file__))


def library_path() -> str:
    return os.path.join(_HERE, "libtilemix.so")


class TilemixError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"tilemix status {status}: {message}")
        self.status = status


class _CParams(ctypes.Structure):
    _fields_ = [
        ("batch", ctypes.c_int32),
        ("heads_q", ctypes.c_int32),
        ("heads_kv", ctypes.c_int32),
        ("len_q", ctypes.c_int32),
        ("len_k", ctypes.c_int32),
        ("head_dim", ctypes.c_int32),
        ("block_m", ctypes.c_int32),
        ("block_n", ctypes.c_int32),
        ("group_size", ctypes.c_int32),
        ("causal", ctypes.c_int32),
        ("scale", ctypes.c_float),
        ("route_per_batch", ctypes.c_int32),
        ("route_hint", ctypes.c_int32),
    ]


@dataclass(frozen=True)
class Params:
    """Mirror of ``tilemix_params``."""
    batch: int
    heads_q: int
    heads_kv: int
    len_q: int
    len_k: int
    head_dim: int
    block_m: int = 128
    block_n: int = 64
    group_size: int = 1
    causal: bool = True
    scale: float = 0.0          # 0 -> 1/sqrt(head_dim)
    route_per_batch: bool = False
    route_hint: int = -1

    def c(self) -> _CParams:
        scale = self.scale if self.scale else 1.0 / math.sqrt(self.head_dim)
        return _CParams(self.batch, self.heads_q, self.heads_kv, self.len_q, self.len_k,
                        self.head_dim, self.block_m, self.block_n, self.group_size,
                        int(bool(self.causal)), scale, int(bool(self.route_per_batch)),
                        self.route_hint)

    @property
    def T_m(self) -> int:
        return -(-self.len_q // self.block_m)

    @property
    def T_n(self) -> int:
        return -(-self.len_k // self.block_n)


TEMPLATE_KINDS = {"one": 0, "zero": 1, "band": 2, "global": 3, "rowrand": 4, "aligned": 5,
                  "bigbird": 6, "sptrans": 7}


class _CTemplate(ctypes.Structure):
    _fields_ = [
        ("kind", ctypes.c_int32),
        ("band_w", ctypes.c_int32),
        ("global_groups", ctypes.c_int32),
        ("rand_fp16", ctypes.c_float),
        ("align_alpha", ctypes.c_float),
        ("align_beta", ctypes.c_float),
        ("sp_stride", ctypes.c_int32),
        ("sp_tail", ctypes.c_int32),
        ("seed", ctypes.c_uint64),
    ]


@dataclass(frozen=True)
class Template:
    """Mirror of ``tilemix_template`` (routing layouts of Appendix B)."""
    kind: str
    band_w: int = 0
    global_groups: int = 0
    rand_fp16: float = 0.0
    align_alpha: float = 0.0
    align_beta: float = 0.0
    sp_stride: int = 0
    sp_tail: int = 0
    seed: int = 0

    def c(self) -> _CTemplate:
        return _CTemplate(TEMPLATE_KINDS[self.kind], self.band_w, self.global_groups, self.rand_fp16,
                          self.align_alpha, self.align_beta, self.sp_stride, self.sp_tail, self.seed)

    @staticmethod
    def from_c(kind: str, t: _CTemplate) -> "Template":
        return Template(kind, t.band_w, t.global_groups, t.rand_fp16, t.align_alpha, t.align_beta,
                        t.sp_stride, t.sp_tail, t.seed)


class _CDebugExport(ctypes.Structure):
    _fields_ = [("q8", ctypes.c_void_p), ("dq", ctypes.c_void_p), ("tiles", ctypes.c_void_p),
                ("kinds", ctypes.c_void_p)]


_LIB = None


def load_library() -> ctypes.CDLL:
    """Load libtilemix.so (raises if it is missing: there is no fallback path).

    torch is imported first: its wheel carries its own HIP runtime under the same soname, and
    the library then binds to that one.  Loaded the other way round, the process would hold two
    HIP runtimes, and the library's would not see the device that torch's owns."""
    global _LIB
    if _LIB is not None:
        return _LIB
    path = library_path()
    if not os.path.exists(path):
        raise RuntimeError(f"{path} is not built; run __graft_entry__.build() first")
    try:
        import torch  # noqa: F401
    except ImportError:  # pragma: no cover - host-only use of the routing templates
        pass
    lib = ctypes.CDLL(path)
    P = ctypes.POINTER(_CParams)
    vp = ctypes.c_void_p
    lib.tilemix_route_words_per_row.argtypes = [P]
    lib.tilemix_route_words_per_row.restype = ctypes.c_int32
    lib.tilemix_workspace_size.argtypes = [P, ctypes.POINTER(ctypes.c_size_t)]
    lib.tilemix_workspace_size.restype = ctypes.c_int
    lib.tilemix_prefill.argtypes = [P, vp, vp, vp, vp, vp, vp, ctypes.c_size_t, vp]
    lib.tilemix_prefill.restype = ctypes.c_int
    lib.tilemix_fused_workspace_size.argtypes = [P, ctypes.POINTER(ctypes.c_size_t)]
    lib.tilemix_fused_workspace_size.restype = ctypes.c_int
    lib.tilemix_prefill_fused.argtypes = [P, vp, vp, vp, vp, vp, vp, ctypes.c_size_t, vp]
    lib.tilemix_prefill_fused.restype = ctypes.c_int
    lib.tilemix_prefill_noalloc.argtypes = [P, vp, vp, vp, vp, vp, vp]
    lib.tilemix_prefill_noalloc.restype = ctypes.c_int
    lib.tilemix_prepare.argtypes = [P, vp, vp, vp, vp, ctypes.c_size_t, vp]
    lib.tilemix_prepare.restype = ctypes.c_int
    lib.tilemix_attend.argtypes = [P, vp, vp, vp, vp, vp, ctypes.c_size_t, vp]
    lib.tilemix_attend.restype = ctypes.c_int
    lib.tilemix_quantize.argtypes = [P, vp, vp, vp, vp, vp, vp, vp]
    lib.tilemix_quantize.restype = ctypes.c_int
    lib.tilemix_debug_qk_int32.argtypes = [P, vp, vp, vp, ctypes.c_int32, vp, vp]
    lib.tilemix_debug_qk_int32.restype = ctypes.c_int
    TP = ctypes.POINTER(_CTemplate)
    lib.tilemix_auto_group_size.argtypes = [ctypes.c_int32, ctypes.c_int32]
    lib.tilemix_auto_group_size.restype = ctypes.c_int32
    lib.tilemix_route_template.argtypes = [P, TP, vp]
    lib.tilemix_route_template.restype = ctypes.c_int
    lib.tilemix_route_template_varlen.argtypes = [P, vp, vp, TP, vp]
    lib.tilemix_route_template_varlen.restype = ctypes.c_int
    lib.tilemix_varlen_workspace_size.argtypes = [P, ctypes.c_int32, ctypes.c_int32,
                                                  ctypes.POINTER(ctypes.c_size_t)]
    lib.tilemix_varlen_workspace_size.restype = ctypes.c_int
    varlen_args = [P, ctypes.c_int32, ctypes.c_int32, vp, vp, vp, vp, vp, vp, ctypes.c_int32, vp, vp,
                   ctypes.c_size_t, vp]
    lib.tilemix_prefill_varlen.argtypes = varlen_args
    lib.tilemix_prefill_varlen.restype = ctypes.c_int
    lib.tilemix_varlen_fused_workspace_size.argtypes = [P, ctypes.c_int32, ctypes.c_int32,
                                                        ctypes.POINTER(ctypes.c_size_t)]
    lib.tilemix_varlen_fused_workspace_size.restype = ctypes.c_int
    lib.tilemix_prefill_varlen_fused.argtypes = varlen_args
    lib.tilemix_prefill_varlen_fused.restype = ctypes.c_int
    lib.tilemix_debug_prefill.argtypes = [P, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32, vp, vp,
                                          vp, vp, vp, vp, ctypes.c_int32, vp, vp, ctypes.c_size_t,
                                          ctypes.POINTER(_CDebugExport), vp]
    lib.tilemix_debug_prefill.restype = ctypes.c_int
    lib.tilemix_quantize_kv.argtypes = [P, vp, vp, vp, vp, vp, vp, vp]
    lib.tilemix_quantize_kv.restype = ctypes.c_int
    lib.tilemix_decode_workspace_size.argtypes = [P, ctypes.POINTER(ctypes.c_size_t)]
    lib.tilemix_decode_workspace_size.restype = ctypes.c_int
    lib.tilemix_decode.argtypes = [P, vp, vp, vp, vp, vp, vp, vp, vp, vp, ctypes.c_size_t, vp]
    lib.tilemix_decode.restype = ctypes.c_int
    lib.tilemix_decode_varlen.argtypes = [P, vp, vp, vp, vp, vp, vp, vp, vp, vp, vp, ctypes.c_size_t, vp]
    lib.tilemix_decode_varlen.restype = ctypes.c_int
    lib.tilemix_route_coverage.argtypes = [P, vp, ctypes.POINTER(ctypes.c_double),
                                           ctypes.POINTER(ctypes.c_double)]
    lib.tilemix_route_coverage.restype = ctypes.c_int
    lib.tilemix_fit_template.argtypes = [P, TP, ctypes.c_double]
    lib.tilemix_fit_template.restype = ctypes.c_int
    lib.tilemix_status_string.argtypes = [ctypes.c_int]
    lib.tilemix_status_string.restype = ctypes.c_char_p
    lib.tilemix_last_error.argtypes = []
    lib.tilemix_last_error.restype = ctypes.c_char_p
    _LIB = lib
    return lib


def _check(status: int) -> None:
    if status != 0:
        lib = load_library()
        msg = lib.tilemix_last_error().decode() or lib.tilemix_status_string(status).decode()
        raise TilemixError(status, msg)


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    import torch
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _alloc(stream, *args, **kw):
    """torch.empty for a buffer the library uses on ``stream``: allocated while that stream is
    current, so that the caching allocator hands the block to no other stream's allocation
    before the work enqueued on ``stream`` is done with it."""
    import torch
    if stream is None:
        return torch.empty(*args, **kw)
    with torch.cuda.stream(stream):
        return torch.empty(*args, **kw)


def tilemix_route_words_per_row(params: Params) -> int:
    return int(load_library().tilemix_route_words_per_row(ctypes.byref(params.c())))


def tilemix_workspace_size(params: Params) -> int:
    n = ctypes.c_size_t(0)
    _check(load_library().tilemix_workspace_size(ctypes.byref(params.c()), ctypes.byref(n)))
    return int(n.value)


def _require(t, dtype, shape, name):
    import torch
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{name} must be a CUDA (HIP) tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if tuple(t.shape) != tuple(shape):
        raise ValueError(f"{name} must have shape {tuple(shape)}, got {tuple(t.shape)}")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")


def _prefill_params(Q, K, group_size, tile, causal, scale, route_per_batch, route_hint) -> Params:
    B, Lq, Hq, d = Q.shape
    Lk, Hk = K.shape[1], K.shape[2]
    return Params(B, Hq, Hk, Lq, Lk, d, tile[0], tile[1], group_size, causal,
                  scale if scale else 1.0 / math.sqrt(d), route_per_batch, route_hint)


def _check_inputs(p: Params, Q, K, V=None):
    import torch
    _require(Q, torch.float16, (p.batch, p.len_q, p.heads_q, p.head_dim), "Q")
    _require(K, torch.float16, (p.batch, p.len_k, p.heads_kv, p.head_dim), "K")
    if V is not None:
        _require(V, torch.float16, (p.batch, p.len_k, p.heads_kv, p.head_dim), "V")


def _workspace(p: Params, workspace, device, fused: bool = False, stream=None, need=None):
    import torch
    if need is None:
        need = tilemix_fused_workspace_size(p) if fused else tilemix_workspace_size(p)
    if workspace is None:
        workspace = _alloc(stream, need, dtype=torch.uint8, device=device)
    nbytes = workspace.numel() * workspace.element_size()
    if nbytes < need:
        raise ValueError(f"workspace too small: {need} bytes needed")
    return workspace, nbytes


def _route_and_out(p: Params, Q, route_bits, O, stream=None):
    import torch
    W = tilemix_route_words_per_row(p)
    _require(route_bits, torch.int64, (p.batch if p.route_per_batch else 1, p.heads_kv, p.T_m, W),
             "route_bits")
    if O is None:
        O = _alloc(stream, (p.batch, p.len_q, p.heads_q, p.head_dim), dtype=torch.float16,
                   device=Q.device)
    _require(O, torch.float16, (p.batch, p.len_q, p.heads_q, p.head_dim), "O")
    return O


def tilemix_prefill(Q, K, V, route_bits, group_size: int, tile=(128, 64), causal: bool = True,
                    scale: float | None = None, *, O=None, workspace=None, stream=None,
                    route_per_batch: bool = False, route_hint: int = -1):
    """Routed prefill attention.  Q [B, Lq, Hq, d], K/V [B, Lk, Hk, d] fp16 CUDA tensors,
    route_bits uint64 words [B_r, Hk, T_m, W] as an int64 CUDA tensor (same bits).
    Returns O (fp16, [B, Lq, Hq, d]).  ``workspace`` (uint8, >= tilemix_workspace_size)
    is allocated when not given."""
    p = _prefill_params(Q, K, group_size, tile, causal, scale, route_per_batch, route_hint)
    _check_inputs(p, Q, K, V)
    O = _route_and_out(p, Q, route_bits, O, stream)
    workspace, nbytes = _workspace(p, workspace, Q.device, stream=stream)
    cp = p.c()
    _check(load_library().tilemix_prefill(
        ctypes.byref(cp), _ptr(Q), _ptr(K), _ptr(V), _ptr(route_bits), _ptr(O), _ptr(workspace),
        ctypes.c_size_t(nbytes), _stream(stream)))
    return O


def tilemix_fused_workspace_size(params: Params) -> int:
    n = ctypes.c_size_t()
    _check(load_library().tilemix_fused_workspace_size(ctypes.byref(params.c()), ctypes.byref(n)))
    return n.value


def tilemix_prefill_fused(Q, K, V, route_bits, group_size: int, tile=(128, 64), causal: bool = True,
                          scale: float | None = None, *, O=None, workspace=None, stream=None,
                          route_per_batch: bool = False, route_hint: int = -1):
    """Routed prefill attention in the fused on-the-fly operand mode (no Q8/K8 scratch; the
    kernel quantizes on chip).  Arguments and result as tilemix_prefill; ``workspace`` (uint8,
    >= tilemix_fused_workspace_size) is allocated when not given."""
    p = _prefill_params(Q, K, group_size, tile, causal, scale, route_per_batch, route_hint)
    _check_inputs(p, Q, K, V)
    O = _route_and_out(p, Q, route_bits, O, stream)
    workspace, nbytes = _workspace(p, workspace, Q.device, fused=True, stream=stream)
    cp = p.c()
    _check(load_library().tilemix_prefill_fused(
        ctypes.byref(cp), _ptr(Q), _ptr(K), _ptr(V), _ptr(route_bits), _ptr(O), _ptr(workspace),
        ctypes.c_size_t(nbytes), _stream(stream)))
    return O


NOALLOC_SCRATCH_BYTES = 128 << 20   # TILEMIX_NOALLOC_SCRATCH_BYTES


def tilemix_prefill_noalloc(Q, K, V, route_bits, group_size: int, tile=(128, 64),
                            causal: bool = True, scale: float | None = None, *, O, stream=None,
                            route_per_batch: bool = False, route_hint: int = -1):
    """tilemix_prefill with no allocation and no workspace argument: the library serves the
    workspace from its own per-GPU device array (at most NOALLOC_SCRATCH_BYTES).  ``O`` is
    required; nothing is allocated here either.  Calls that overlap on one GPU race."""
    p = _prefill_params(Q, K, group_size, tile, causal, scale, route_per_batch, route_hint)
    _check_inputs(p, Q, K, V)
    O = _route_and_out(p, Q, route_bits, O, stream)
    cp = p.c()
    _check(load_library().tilemix_prefill_noalloc(
        ctypes.byref(cp), _ptr(Q), _ptr(K), _ptr(V), _ptr(route_bits), _ptr(O), _stream(stream)))
    return O


def tilemix_prepare(Q, K, V, group_size: int, tile=(128, 64), causal: bool = True,
                    scale: float | None = None, *, workspace=None, stream=None,
                    route_per_batch: bool = False, route_hint: int = -1):
    """Operand preparation (quantize-once + V tile layout) into ``workspace``; returns it."""
    p = _prefill_params(Q, K, group_size, tile, causal, scale, route_per_batch, route_hint)
    _check_inputs(p, Q, K, V)
    workspace, nbytes = _workspace(p, workspace, Q.device, stream=stream)
    cp = p.c()
    _check(load_library().tilemix_prepare(ctypes.byref(cp), _ptr(Q), _ptr(K), _ptr(V), _ptr(workspace),
                                          ctypes.c_size_t(nbytes), _stream(stream)))
    return workspace


def tilemix_attend(Q, K, route_bits, workspace, group_size: int, tile=(128, 64), causal: bool = True,
                   scale: float | None = None, *, O=None, stream=None, route_per_batch: bool = False,
                   route_hint: int = -1):
    """Fused routed attention on a workspace filled by tilemix_prepare; returns O."""
    p = _prefill_params(Q, K, group_size, tile, causal, scale, route_per_batch, route_hint)
    _check_inputs(p, Q, K)
    O = _route_and_out(p, Q, route_bits, O, stream)
    workspace, nbytes = _workspace(p, workspace, Q.device, stream=stream)
    cp = p.c()
    _check(load_library().tilemix_attend(ctypes.byref(cp), _ptr(Q), _ptr(K), _ptr(route_bits), _ptr(O),
                                         _ptr(workspace), ctypes.c_size_t(nbytes), _stream(stream)))
    return O


def tilemix_quantize(Q, K, *, tile=(128, 64), stream=None):
    """Quantize-once pass.  Returns (Q8 int8, dQ fp16, K8 int8, dK fp16) CUDA tensors."""
    import torch
    B, Lq, Hq, d = Q.shape
    Lk, Hk = K.shape[1], K.shape[2]
    p = Params(B, Hq, Hk, Lq, Lk, d, tile[0], tile[1])
    _require(Q, torch.float16, (B, Lq, Hq, d), "Q")
    _require(K, torch.float16, (B, Lk, Hk, d), "K")
    Q8 = _alloc(stream, (B, Lq, Hq, d), dtype=torch.int8, device=Q.device)
    K8 = _alloc(stream, (B, Lk, Hk, d), dtype=torch.int8, device=Q.device)
    dQ = _alloc(stream, (B, -(-Lq // 128), Hq), dtype=torch.float16, device=Q.device)
    dK = _alloc(stream, (B, -(-Lk // 64), Hk), dtype=torch.float16, device=Q.device)
    cp = p.c()
    _check(load_library().tilemix_quantize(ctypes.byref(cp), _ptr(Q), _ptr(K), _ptr(Q8), _ptr(dQ),
                                           _ptr(K8), _ptr(dK), _stream(stream)))
    return Q8, dQ, K8, dK


def tilemix_debug_qk_int32(Q8, K8, tiles, *, heads_q: int, heads_kv: int, tile=(128, 64),
                           stream=None):
    """INT32 tile products for rows (b, h_q, m, n) of ``tiles`` (int32 CUDA [count, 4]).
    Returns int32 [count, BLOCK_M, BLOCK_N]."""
    import torch
    B, Lq, Hq, d = Q8.shape
    Lk = K8.shape[1]
    p = Params(B, heads_q, heads_kv, Lq, Lk, d, tile[0], tile[1])
    _require(Q8, torch.int8, (B, Lq, heads_q, d), "Q8")
    _require(K8, torch.int8, (B, Lk, heads_kv, d), "K8")
    count = tiles.shape[0]
    _require(tiles, torch.int32, (count, 4), "tiles")
    out = _alloc(stream, (count, tile[0], tile[1]), dtype=torch.int32, device=Q8.device)
    cp = p.c()
    _check(load_library().tilemix_debug_qk_int32(ctypes.byref(cp), _ptr(Q8), _ptr(K8), _ptr(tiles),
                                                 ctypes.c_int32(count), _ptr(out), _stream(stream)))
    return out


# ----------------------------------------------------------------- routing templates (host)

def tilemix_auto_group_size(len_k: int, block_n: int = 64) -> int:
    """The paper's automatic routing-group size g for L_k keys (0 if an argument is < 1)."""
    return int(load_library().tilemix_auto_group_size(len_k, block_n))


def _host_words_shape(p: Params):
    return (p.batch if p.route_per_batch else 1, p.heads_kv, p.T_m, tilemix_route_words_per_row(p))


def tilemix_route_template(params: Params, template: Template):
    """Routing words (host NumPy uint64 [B_r, H_k, T_m, W]) of ``template`` for ``params``."""
    import numpy as np
    shape = _host_words_shape(params)
    words = np.zeros(shape, dtype=np.uint64)
    cp, ct = params.c(), template.c()
    _check(load_library().tilemix_route_template(ctypes.byref(cp), ctypes.byref(ct),
                                                 words.ctypes.data_as(ctypes.c_void_p)))
    return words


def tilemix_route_coverage(params: Params, words):
    """(rho_groups, rho_pairs): realized INT8 coverage of host routing words."""
    import numpy as np
    w = np.ascontiguousarray(words, dtype=np.uint64)
    if w.shape != _host_words_shape(params):
        raise ValueError(f"words must have shape {_host_words_shape(params)}, got {w.shape}")
    rg, rp = ctypes.c_double(0.0), ctypes.c_double(0.0)
    cp = params.c()
    _check(load_library().tilemix_route_coverage(ctypes.byref(cp), w.ctypes.data_as(ctypes.c_void_p),
                                                 ctypes.byref(rg), ctypes.byref(rp)))
    return rg.value, rp.value


def tilemix_fit_template(params: Params, template: Template, rho_int8: float) -> Template:
    """The template with its size parameter chosen to match INT8 coverage ``rho_int8``."""
    cp, ct = params.c(), template.c()
    _check(load_library().tilemix_fit_template(ctypes.byref(cp), ctypes.byref(ct),
                                               ctypes.c_double(rho_int8)))
    return Template.from_c(template.kind, ct)


def tilemix_route_template_varlen(params: Params, seqlens_q, seqlens_k, template: Template):
    """Routing words (host uint64 [sum_b ceil(L_q,b / BLOCK_M), H_k, W]) of ``template`` for each
    sequence of a variable-length batch (``params.len_q``/``len_k`` = maximum lengths)."""
    import numpy as np
    lq = np.ascontiguousarray(seqlens_q, dtype=np.int32)
    lk = np.ascontiguousarray(seqlens_k, dtype=np.int32)
    if lq.shape != (params.batch,) or lk.shape != (params.batch,):
        raise ValueError("seqlens_q / seqlens_k must have one entry per sequence")
    rows = int(sum(-(-int(x) // params.block_m) for x in lq))
    words = np.zeros((rows, params.heads_kv, tilemix_route_words_per_row(params)), dtype=np.uint64)
    cp, ct = params.c(), template.c()
    _check(load_library().tilemix_route_template_varlen(
        ctypes.byref(cp), lq.ctypes.data_as(ctypes.c_void_p), lk.ctypes.data_as(ctypes.c_void_p),
        ctypes.byref(ct), words.ctypes.data_as(ctypes.c_void_p)))
    return words


def tilemix_varlen_workspace_size(params: Params, total_q: int, total_k: int) -> int:
    n = ctypes.c_size_t(0)
    _check(load_library().tilemix_varlen_workspace_size(ctypes.byref(params.c()), total_q, total_k,
                                                        ctypes.byref(n)))
    return int(n.value)


def tilemix_varlen_fused_workspace_size(params: Params, total_q: int, total_k: int) -> int:
    n = ctypes.c_size_t(0)
    _check(load_library().tilemix_varlen_fused_workspace_size(ctypes.byref(params.c()), total_q,
                                                              total_k, ctypes.byref(n)))
    return int(n.value)


def _varlen_call(name, Q, K, V, cu_seqlens_q, cu_seqlens_k, max_len_q, max_len_k, route_bits,
                 group_size, tile, causal, scale, O, workspace, stream, route_hint, fused):
    import torch
    total_q, Hq, d = Q.shape
    total_k, Hk = K.shape[0], K.shape[1]
    B = cu_seqlens_q.shape[0] - 1
    p = Params(B, Hq, Hk, max_len_q, max_len_k, d, tile[0], tile[1], group_size, causal,
               scale if scale else 1.0 / math.sqrt(d), False, route_hint)
    _require(Q, torch.float16, (total_q, Hq, d), "Q")
    _require(K, torch.float16, (total_k, Hk, d), "K")
    _require(V, torch.float16, (total_k, Hk, d), "V")
    _require(cu_seqlens_q, torch.int32, (B + 1,), "cu_seqlens_q")
    _require(cu_seqlens_k, torch.int32, (B + 1,), "cu_seqlens_k")
    if route_bits.dim() != 3 or tuple(route_bits.shape[1:]) != (Hk, tilemix_route_words_per_row(p)):
        raise ValueError("route_bits must be [rows, H_k, W]")
    _require(route_bits, torch.int64, tuple(route_bits.shape), "route_bits")
    if O is None:
        O = _alloc(stream, (total_q, Hq, d), dtype=torch.float16, device=Q.device)
    _require(O, torch.float16, (total_q, Hq, d), "O")
    need = (tilemix_varlen_fused_workspace_size(p, total_q, total_k) if fused
            else tilemix_varlen_workspace_size(p, total_q, total_k))
    workspace, nbytes = _workspace(p, workspace, Q.device, stream=stream, need=need)
    cp = p.c()
    _check(getattr(load_library(), name)(
        ctypes.byref(cp), total_q, total_k, _ptr(cu_seqlens_q), _ptr(cu_seqlens_k), _ptr(Q), _ptr(K),
        _ptr(V), _ptr(route_bits), ctypes.c_int32(route_bits.shape[0]), _ptr(O), _ptr(workspace),
        ctypes.c_size_t(nbytes), _stream(stream)))
    return O


def tilemix_prefill_varlen(Q, K, V, cu_seqlens_q, cu_seqlens_k, max_len_q: int, max_len_k: int,
                           route_bits, group_size: int, tile=(128, 64), causal: bool = True,
                           scale: float | None = None, *, O=None, workspace=None, stream=None,
                           route_hint: int = -1):
    """Routed prefill attention over a packed variable-length batch.  Q [total_q, Hq, d],
    K/V [total_k, Hk, d] fp16 CUDA tensors; cu_seqlens_q/k int32 CUDA [B + 1]; route_bits the
    uint64 words [sum_b ceil(L_q,b / BLOCK_M), Hk, W] as an int64 CUDA tensor.  Returns O."""
    return _varlen_call("tilemix_prefill_varlen", Q, K, V, cu_seqlens_q, cu_seqlens_k, max_len_q,
                        max_len_k, route_bits, group_size, tile, causal, scale, O, workspace, stream,
                        route_hint, False)


def tilemix_prefill_varlen_fused(Q, K, V, cu_seqlens_q, cu_seqlens_k, max_len_q: int,
                                 max_len_k: int, route_bits, group_size: int, tile=(128, 64),
                                 causal: bool = True, scale: float | None = None, *, O=None,
                                 workspace=None, stream=None, route_hint: int = -1):
    """tilemix_prefill_varlen in the fused on-the-fly operand mode (no K8 / scale tensors)."""
    return _varlen_call("tilemix_prefill_varlen_fused", Q, K, V, cu_seqlens_q, cu_seqlens_k,
                        max_len_q, max_len_k, route_bits, group_size, tile, causal, scale, O,
                        workspace, stream, route_hint, True)


def tilemix_debug_prefill(Q, K, V, route_bits, group_size: int, tile=(128, 64), causal: bool = True,
                          scale: float | None = None, *, fused: bool = False, cu_seqlens_q=None,
                          cu_seqlens_k=None, max_len_q: int = 0, max_len_k: int = 0,
                          route_per_batch: bool = False, route_hint: int = -1, stream=None):
    """Test entry point: one prefill call (fixed-length [B, L, H, d] inputs, or packed
    [total, H, d] ones with ``cu_seqlens_q/k`` and the maximum lengths) whose kernel also exports
    the INT8 operands it made and multiplied.  Returns (O, q8, dq, tiles, kinds): q8 like Q
    (pre-filled with -128), dq int16 bits [R, Hq] (pre-filled with -1), tiles int32
    [R, Hq, T_n, BLOCK_M, 64] and kinds int32 [R, Hq, T_n, BLOCK_M // 32] (pre-filled with 0),
    R the query-tile rows (B * T_m, or the rows of ``route_bits`` for a packed batch)."""
    import torch
    varlen = cu_seqlens_q is not None
    if varlen:
        total_q, Hq, d = Q.shape
        total_k, Hk = K.shape[0], K.shape[1]
        B = cu_seqlens_q.shape[0] - 1
        p = Params(B, Hq, Hk, max_len_q, max_len_k, d, tile[0], tile[1], group_size, causal,
                   scale if scale else 1.0 / math.sqrt(d), False, route_hint)
        _require(Q, torch.float16, (total_q, Hq, d), "Q")
        _require(K, torch.float16, (total_k, Hk, d), "K")
        _require(V, torch.float16, (total_k, Hk, d), "V")
        _require(cu_seqlens_q, torch.int32, (B + 1,), "cu_seqlens_q")
        _require(cu_seqlens_k, torch.int32, (B + 1,), "cu_seqlens_k")
        if route_bits.dim() != 3 or tuple(route_bits.shape[1:]) != (Hk, tilemix_route_words_per_row(p)):
            raise ValueError("route_bits must be [rows, H_k, W]")
        _require(route_bits, torch.int64, tuple(route_bits.shape), "route_bits")
        rows = route_bits.shape[0]
        O = _alloc(stream, (total_q, Hq, d), dtype=torch.float16, device=Q.device)
        need = (tilemix_varlen_fused_workspace_size(p, total_q, total_k) if fused
                else tilemix_varlen_workspace_size(p, total_q, total_k))
    else:
        p = _prefill_params(Q, K, group_size, tile, causal, scale, route_per_batch, route_hint)
        _check_inputs(p, Q, K, V)
        O = _route_and_out(p, Q, route_bits, None, stream)
        total_q = total_k = -1
        rows = p.batch * p.T_m
        need = tilemix_fused_workspace_size(p) if fused else tilemix_workspace_size(p)
    workspace, nbytes = _workspace(p, None, Q.device, stream=stream, need=need)
    q8 = _alloc(stream, tuple(Q.shape), dtype=torch.int8, device=Q.device)
    dq = _alloc(stream, (rows, p.heads_q), dtype=torch.int16, device=Q.device)
    tiles = _alloc(stream, (rows, p.heads_q, p.T_n, p.block_m, 64), dtype=torch.int32, device=Q.device)
    kinds = _alloc(stream, (rows, p.heads_q, p.T_n, p.block_m // 32), dtype=torch.int32,
                   device=Q.device)
    with torch.cuda.stream(stream if stream is not None else torch.cuda.current_stream()):
        q8.fill_(-128)
        dq.fill_(-1)
        tiles.zero_()
        kinds.zero_()
    exp = _CDebugExport(_ptr(q8), _ptr(dq), _ptr(tiles), _ptr(kinds))
    cp = p.c()
    _check(load_library().tilemix_debug_prefill(
        ctypes.byref(cp), int(bool(fused)), total_q, total_k, _ptr(cu_seqlens_q), _ptr(cu_seqlens_k),
        _ptr(Q), _ptr(K), _ptr(V), _ptr(route_bits), ctypes.c_int32(rows if varlen else 0), _ptr(O),
        _ptr(workspace), ctypes.c_size_t(nbytes), ctypes.byref(exp), _stream(stream)))
    return O, q8, dq, tiles, kinds


# ------------------------------------------------------------ INT8 key/value cache decode

def tilemix_quantize_kv(K, V, *, stream=None):
    """INT8 key/value cache of K, V [B, L_k, H_k, d] (fp16 CUDA): (K8, dK, V8, dV) with K8
    [B, L_k, H_k, d] and V8 [B, H_k, ceil(L_k/64), d, 64] (each 64-key block channel-major)."""
    import torch
    B, Lk, Hk, d = K.shape
    p = Params(B, Hk, Hk, 1, Lk, d)
    _require(K, torch.float16, (B, Lk, Hk, d), "K")
    _require(V, torch.float16, (B, Lk, Hk, d), "V")
    K8 = _alloc(stream, (B, Lk, Hk, d), dtype=torch.int8, device=K.device)
    V8 = _alloc(stream, (B, Hk, -(-Lk // 64), d, 64), dtype=torch.int8, device=K.device)
    dK = _alloc(stream, (B, -(-Lk // 64), Hk), dtype=torch.float16, device=K.device)
    dV = _alloc(stream, (B, -(-Lk // 64), Hk), dtype=torch.float16, device=K.device)
    cp = p.c()
    _check(load_library().tilemix_quantize_kv(ctypes.byref(cp), _ptr(K), _ptr(V), _ptr(K8), _ptr(dK),
                                              _ptr(V8), _ptr(dV), _stream(stream)))
    return K8, dK, V8, dV


def tilemix_decode_workspace_size(params: Params) -> int:
    n = ctypes.c_size_t(0)
    _check(load_library().tilemix_decode_workspace_size(ctypes.byref(params.c()), ctypes.byref(n)))
    return int(n.value)


def tilemix_decode(Q, K, K8, dK, V8, dV, route_bits, group_size: int, scale: float | None = None,
                   *, O=None, workspace=None, stream=None, route_per_batch: bool = False,
                   route_hint: int = -1, seqlens_k=None):
    """One decode step: Q [B, 1, Hq, d] against the FP16 key cache K [B, L_k, H_k, d] and the
    INT8 caches of tilemix_quantize_kv; route_bits int64 CUDA [B_r, H_k, 1, W].  Returns O.
    With ``seqlens_k`` (int32 CUDA [B]) sequence b uses its first seqlens_k[b] cached keys
    (tilemix_decode_varlen; L_k is then the caches' capacity)."""
    import torch
    B, Lq, Hq, d = Q.shape
    Lk, Hk = K.shape[1], K.shape[2]
    p = Params(B, Hq, Hk, Lq, Lk, d, 128, 64, group_size, True,
               scale if scale else 1.0 / math.sqrt(d), route_per_batch, route_hint)
    _require(Q, torch.float16, (B, 1, Hq, d), "Q")
    _require(K, torch.float16, (B, Lk, Hk, d), "K")
    _require(K8, torch.int8, (B, Lk, Hk, d), "K8")
    _require(V8, torch.int8, (B, Hk, -(-Lk // 64), d, 64), "V8")
    _require(dK, torch.float16, (B, -(-Lk // 64), Hk), "dK")
    _require(dV, torch.float16, (B, -(-Lk // 64), Hk), "dV")
    _require(route_bits, torch.int64, (B if route_per_batch else 1, Hk, 1, tilemix_route_words_per_row(p)),
             "route_bits")
    if O is None:
        O = _alloc(stream, tuple(Q.shape), dtype=torch.float16, device=Q.device)
    _require(O, torch.float16, (B, 1, Hq, d), "O")
    workspace, nbytes = _workspace(p, workspace, Q.device, stream=stream,
                                   need=tilemix_decode_workspace_size(p))
    cp = p.c()
    if seqlens_k is not None:
        _require(seqlens_k, torch.int32, (B,), "seqlens_k")
        _check(load_library().tilemix_decode_varlen(
            ctypes.byref(cp), _ptr(seqlens_k), _ptr(Q), _ptr(K), _ptr(K8), _ptr(dK), _ptr(V8),
            _ptr(dV), _ptr(route_bits), _ptr(O), _ptr(workspace), ctypes.c_size_t(nbytes),
            _stream(stream)))
        return O
    _check(load_library().tilemix_decode(ctypes.byref(cp), _ptr(Q), _ptr(K), _ptr(K8), _ptr(dK), _ptr(V8),
                                         _ptr(dV), _ptr(route_bits), _ptr(O), _ptr(workspace),
                                         ctypes.c_size_t(nbytes), _stream(stream)))
    return O
