"""ctypes binding of the C-ABI (argument marshalling only).

Functions carry the C names without the ``mc_`` prefix.  Device buffers are
torch tensors on the current CUDA (HIP) device; the library never allocates,
so ``PackedLayer`` and ``Routing`` allocate their buffers with torch and build
the descriptors over them.
"""
from __future__ import annotations

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "libmcmoe.so")
_lib = None

MC_OK, MC_EINVAL, MC_ENOSPACE, MC_EHIP, MC_EUNSUPPORTED = range(5)
MAX_EXPERTS = 256
MAX_TOPK = 8


class MCError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__("mc status %d: %s" % (status, msg))
        self.status = status


class _Layer(ctypes.Structure):
    _fields_ = [("E", ctypes.c_int), ("d", ctypes.c_int), ("ffn", ctypes.c_int),
                ("group", ctypes.c_int), ("bits_host", ctypes.POINTER(ctypes.c_int)),
                ("words", ctypes.c_void_p), ("sz", ctypes.c_void_p),
                ("words_bytes", ctypes.c_size_t), ("sz_bytes", ctypes.c_size_t)]


class _Routing(ctypes.Structure):
    _fields_ = [("T", ctypes.c_int), ("E", ctypes.c_int), ("k", ctypes.c_int),
                ("topk_idx", ctypes.c_void_p), ("topk_w", ctypes.c_void_p),
                ("kept", ctypes.c_void_p), ("counts", ctypes.c_void_p),
                ("offsets", ctypes.c_void_p), ("pair_token", ctypes.c_void_p),
                ("pair_rank", ctypes.c_void_p), ("pair_w", ctypes.c_void_p),
                ("pair_pos", ctypes.c_void_p), ("n_pruned", ctypes.c_void_p)]


def lib_path() -> str:
    return _LIB_PATH


def load():
    """Load libmcmoe.so; raises if it has not been built."""
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            raise RuntimeError("libmcmoe.so is not built (run __graft_entry__.build())")
        lib = ctypes.CDLL(_LIB_PATH)
        P, I, S = ctypes.c_void_p, ctypes.c_int, ctypes.c_size_t
        st = ctypes.c_int
        lib.mc_last_error.restype = ctypes.c_char_p
        lib.mc_last_error.argtypes = []
        lib.mc_pack_sizes.restype = st
        lib.mc_pack_sizes.argtypes = [I, I, I, P, I, ctypes.POINTER(S), ctypes.POINTER(S)]
        lib.mc_pack.restype = st
        lib.mc_pack.argtypes = [P, P, P, ctypes.POINTER(_Layer), P]
        lib.mc_pack_methods.restype = st
        lib.mc_pack_methods.argtypes = [P, P, P, ctypes.POINTER(_Layer), P, P]
        lib.mc_dequant_export.restype = st
        lib.mc_dequant_export.argtypes = [ctypes.POINTER(_Layer), I, I, P, P]
        lib.mc_codes_export.restype = st
        lib.mc_codes_export.argtypes = [ctypes.POINTER(_Layer), I, I, P, P]
        lib.mc_gptq_workspace.restype = st
        lib.mc_gptq_workspace.argtypes = [I, I, ctypes.POINTER(S)]
        lib.mc_gptq_hessian.restype = st
        lib.mc_gptq_hessian.argtypes = [P, I, I, P, I, P]
        lib.mc_gptq_factor.restype = st
        lib.mc_gptq_factor.argtypes = [P, I, ctypes.c_double, P, P, P, S, P]
        lib.mc_gptq_quantize.restype = st
        lib.mc_gptq_quantize.argtypes = [ctypes.POINTER(_Layer), I, I, P, P, P, P, P, S, P]
        lib.mc_router_logits.restype = st
        lib.mc_router_logits.argtypes = [P, P, I, I, I, P, P]
        lib.mc_route_and_prune.restype = st
        lib.mc_route_and_prune.argtypes = [P, P, ctypes.c_float, ctypes.POINTER(_Routing), P]
        lib.mc_forward_workspace.restype = st
        lib.mc_forward_workspace.argtypes = [I, I, I, I, I, ctypes.POINTER(S)]
        lib.mc_moe_forward.restype = st
        lib.mc_moe_forward.argtypes = [P, ctypes.POINTER(_Routing), ctypes.POINTER(_Layer), P, P,
                                       S, P]
        lib.mc_moe_forward_noalloc.restype = st
        lib.mc_moe_forward_noalloc.argtypes = [P, ctypes.POINTER(_Routing), ctypes.POINTER(_Layer), P, P]
        lib.mc_moe_route_forward.restype = st
        lib.mc_moe_route_forward.argtypes = [P, P, P, ctypes.c_float, ctypes.POINTER(_Routing),
                                             ctypes.POINTER(_Layer), P, P, S, P]
        lib.mc_stack_workspace.restype = st
        lib.mc_stack_workspace.argtypes = [I, I, I, I, I, ctypes.POINTER(S)]
        lib.mc_moe_stack_forward.restype = st
        lib.mc_moe_stack_forward.argtypes = [P, I, ctypes.POINTER(_Layer), P, P, ctypes.c_float,
                                             ctypes.POINTER(_Routing), P, P, P, S, P]
        lib.mc_importance_workspace.restype = st
        lib.mc_importance_workspace.argtypes = [I, I, ctypes.POINTER(S)]
        lib.mc_token_importance.restype = st
        lib.mc_token_importance.argtypes = [P, I, I, P, I, ctypes.c_float, P, P, P, S, P]
        lib.mc_odp_threshold.restype = st
        lib.mc_odp_threshold.argtypes = [P, I, I, ctypes.POINTER(ctypes.c_double),
                                         ctypes.POINTER(ctypes.c_double)]
        D = ctypes.c_double
        lib.mc_pmq_significance.restype = st
        lib.mc_pmq_significance.argtypes = [P, I, I, I, P, P]
        lib.mc_pmq_allocate.restype = st
        lib.mc_pmq_allocate.argtypes = [P, P, P, I, D, D, D, I, P, ctypes.POINTER(D)]
        lib.mc_pmq_error_workspace.restype = st
        lib.mc_pmq_error_workspace.argtypes = [I, I, I, I, I, I, ctypes.POINTER(S)]
        lib.mc_pmq_expert_error.restype = st
        lib.mc_pmq_expert_error.argtypes = [P, P, P, I, I, I, I, P, ctypes.POINTER(_Routing), P, P, S, P]
        lib.mc_timing_enable.restype = st
        lib.mc_timing_enable.argtypes = [I]
        lib.mc_timing_read.restype = st
        lib.mc_timing_read.argtypes = [ctypes.c_char_p, ctypes.POINTER(ctypes.c_double),
                                       ctypes.POINTER(I)]
        _lib = lib
    return _lib


def _check(status: int):
    if status != MC_OK:
        raise MCError(status, load().mc_last_error().decode())


def _stream(stream=None):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def pack_sizes(E: int, d: int, ffn: int, bits, group: int):
    arr = (ctypes.c_int * len(bits))(*[int(b) for b in bits])
    wb, szb = ctypes.c_size_t(), ctypes.c_size_t()
    _check(load().mc_pack_sizes(E, d, ffn, arr, group, ctypes.byref(wb), ctypes.byref(szb)))
    return wb.value, szb.value


class PackedLayer:
    """Device buffers + descriptor of one packed layer (torch-allocated)."""

    def __init__(self, E: int, d: int, ffn: int, bits, group: int, device=None):
        self.E, self.d, self.ffn, self.group = E, d, ffn, group
        self.bits = [int(b) for b in bits]
        wb, szb = pack_sizes(E, d, ffn, self.bits, group)
        device = device or torch.device("cuda")
        self.words = torch.empty(wb // 4, dtype=torch.int32, device=device)
        self.sz = torch.empty(szb // 4, dtype=torch.int32, device=device)
        self._bits_c = (ctypes.c_int * E)(*self.bits)
        self.desc = _Layer(E, d, ffn, group, self._bits_c, self.words.data_ptr(),
                           self.sz.data_ptr(), wb, szb)

    @property
    def nbytes(self) -> int:
        return self.words.numel() * 4 + self.sz.numel() * 4


class Routing:
    """Device buffers + descriptor of a routing result for T tokens."""

    def __init__(self, T: int, E: int, k: int, device=None):
        device = device or torch.device("cuda")
        self.T, self.E, self.k = T, E, k
        i32 = dict(dtype=torch.int32, device=device)
        self.topk_idx = torch.empty((T, k), **i32)
        self.topk_w = torch.empty((T, k), dtype=torch.float32, device=device)
        self.kept = torch.empty((T, k), dtype=torch.uint8, device=device)
        self.counts = torch.empty(E, **i32)
        self.offsets = torch.empty(E + 1, **i32)
        self.pair_token = torch.full((T * k,), -1, **i32)
        self.pair_rank = torch.full((T * k,), -1, **i32)
        self.pair_w = torch.zeros(T * k, dtype=torch.float32, device=device)
        self.pair_pos = torch.empty((T, k), **i32)
        self.n_pruned = torch.empty(1, **i32)
        self.desc = _Routing(T, E, k, *[t.data_ptr() for t in (
            self.topk_idx, self.topk_w, self.kept, self.counts, self.offsets, self.pair_token,
            self.pair_rank, self.pair_w, self.pair_pos, self.n_pruned)])


QUANT_RTN, QUANT_SIGN = 0, 1


def pack(w_gate, w_up, w_down, layer: PackedLayer, stream=None, methods=None):
    """Quantize and pack; methods (per expert, QUANT_RTN or QUANT_SIGN for
    1-bit sign binarization) defaults to RTN everywhere."""
    for t in (w_gate, w_up, w_down):
        assert t.dtype == torch.float32 and t.is_contiguous() and t.is_cuda
    if methods is None:
        _check(load().mc_pack(_ptr(w_gate), _ptr(w_up), _ptr(w_down), ctypes.byref(layer.desc),
                              _stream(stream)))
    else:
        arr = (ctypes.c_int * layer.E)(*[int(m) for m in methods])
        _check(load().mc_pack_methods(_ptr(w_gate), _ptr(w_up), _ptr(w_down), ctypes.byref(layer.desc),
                                      arr, _stream(stream)))


def dequant_export(layer: PackedLayer, e: int, mat: int, out, stream=None):
    assert out.dtype in (torch.float16, torch.int16) and out.is_contiguous()
    _check(load().mc_dequant_export(ctypes.byref(layer.desc), e, mat, _ptr(out), _stream(stream)))


def codes_export(layer: PackedLayer, e: int, mat: int, out, stream=None):
    assert out.dtype == torch.uint8 and out.is_contiguous()
    _check(load().mc_codes_export(ctypes.byref(layer.desc), e, mat, _ptr(out), _stream(stream)))


def gptq_workspace(R: int, K: int) -> int:
    b = ctypes.c_size_t()
    _check(load().mc_gptq_workspace(R, K, ctypes.byref(b)))
    return b.value


def gptq_hessian(x, H, accumulate: bool = False, stream=None):
    """x: [N][K] bf16 (or int16 bits); H: [K][K] float64."""
    assert x.is_contiguous() and x.element_size() == 2 and H.is_contiguous() and H.dtype == torch.float64
    N, K = x.shape
    assert tuple(H.shape) == (K, K)
    _check(load().mc_gptq_hessian(_ptr(x), N, K, _ptr(H), int(bool(accumulate)), _stream(stream)))


def gptq_factor(H, U, dead, workspace, damp: float = 0.01, stream=None):
    """H, U: [K][K] float64; dead: [K] uint8."""
    K = H.shape[0]
    assert H.is_contiguous() and U.is_contiguous() and H.dtype == torch.float64 and U.dtype == torch.float64
    assert dead.dtype == torch.uint8 and dead.numel() == K
    _check(load().mc_gptq_factor(_ptr(H), K, float(damp), _ptr(U), _ptr(dead), _ptr(workspace),
                                 workspace.numel() * workspace.element_size(), _stream(stream)))


def gptq_quantize(layer: PackedLayer, e: int, mat: int, W, U, dead, workspace, loss=None, stream=None):
    """W: [R][K] float32 (the fp32 weights of matrix `mat` of expert e)."""
    assert W.is_contiguous() and W.dtype == torch.float32 and U.dtype == torch.float64
    _check(load().mc_gptq_quantize(ctypes.byref(layer.desc), e, mat, _ptr(W), _ptr(U), _ptr(dead), _ptr(loss),
                                   _ptr(workspace), workspace.numel() * workspace.element_size(),
                                   _stream(stream)))


def router_logits(x, w_router, logits, stream=None):
    """x [T][d], w_router [E][d]: bf16 (or int16 bit patterns); logits [T][E] fp32."""
    assert x.is_contiguous() and w_router.is_contiguous() and logits.is_contiguous()
    assert x.element_size() == 2 and w_router.element_size() == 2 and logits.dtype == torch.float32
    T, d = x.shape
    E = w_router.shape[0]
    assert w_router.shape[1] == d and tuple(logits.shape) == (T, E)
    _check(load().mc_router_logits(_ptr(x), _ptr(w_router), T, d, E, _ptr(logits), _stream(stream)))


def route_and_prune(logits, important, threshold: float, routing: Routing, stream=None):
    assert logits.dtype == torch.float32 and logits.is_contiguous()
    if important is not None:
        assert important.dtype == torch.uint8 and important.is_contiguous()
    _check(load().mc_route_and_prune(_ptr(logits), _ptr(important), float(threshold),
                                     ctypes.byref(routing.desc), _stream(stream)))


def forward_workspace(T: int, E: int, k: int, d: int, ffn: int) -> int:
    b = ctypes.c_size_t()
    _check(load().mc_forward_workspace(T, E, k, d, ffn, ctypes.byref(b)))
    return b.value


def moe_forward(x, routing: Routing, layer: PackedLayer, y, workspace, stream=None):
    """x, y: bf16 (or int16 bit patterns) [T][d] device tensors."""
    assert x.is_contiguous() and y.is_contiguous() and x.element_size() == 2
    _check(load().mc_moe_forward(_ptr(x), ctypes.byref(routing.desc), ctypes.byref(layer.desc),
                                 _ptr(y), _ptr(workspace), workspace.numel() * workspace.element_size(),
                                 _stream(stream)))


def moe_forward_noalloc(x, routing: Routing, layer: PackedLayer, y, stream=None):
    """moe_forward with the library's own device workspace (no allocation)."""
    assert x.is_contiguous() and y.is_contiguous() and x.element_size() == 2
    _check(load().mc_moe_forward_noalloc(_ptr(x), ctypes.byref(routing.desc), ctypes.byref(layer.desc),
                                         _ptr(y), _stream(stream)))


def route_forward(x, logits, important, threshold: float, routing: Routing, layer: PackedLayer, y, workspace,
                  stream=None):
    """route_and_prune + moe_forward in one call (same results)."""
    assert x.is_contiguous() and y.is_contiguous() and x.element_size() == 2
    assert logits.dtype == torch.float32 and logits.is_contiguous()
    if important is not None:
        assert important.dtype == torch.uint8 and important.is_contiguous()
    _check(load().mc_moe_route_forward(_ptr(x), _ptr(logits), _ptr(important), float(threshold),
                                       ctypes.byref(routing.desc), ctypes.byref(layer.desc), _ptr(y),
                                       _ptr(workspace), workspace.numel() * workspace.element_size(),
                                       _stream(stream)))


def stack_workspace(T: int, E: int, k: int, d: int, ffn: int) -> int:
    b = ctypes.c_size_t()
    _check(load().mc_stack_workspace(T, E, k, d, ffn, ctypes.byref(b)))
    return b.value


def stack_forward(x, layers, logits, important, threshold: float, routing: Routing, y, tmp,
                  workspace, stream=None):
    """Residual MoE stack: y = h_n with h_{l+1} = bf16(h_l + MoE_l(RMSNorm(h_l))).
    x, y, tmp: bf16 bits [T][d]; logits: float32 [n][T][E]; important: uint8
    [n][T] or None; layers: list of PackedLayer sharing E, d, ffn, group."""
    n = len(layers)
    arr = (_Layer * n)(*[l.desc for l in layers])
    assert logits.dtype == torch.float32 and logits.is_contiguous()
    for t in (x, y) + (() if tmp is None else (tmp,)):
        assert t.is_contiguous() and t.element_size() == 2
    _check(load().mc_moe_stack_forward(_ptr(x), n, arr, _ptr(logits), _ptr(important),
                                       float(threshold), ctypes.byref(routing.desc), _ptr(y), _ptr(tmp),
                                       _ptr(workspace), workspace.numel() * workspace.element_size(),
                                       _stream(stream)))


def importance_workspace(H: int, L: int) -> int:
    b = ctypes.c_size_t()
    _check(load().mc_importance_workspace(H, L, ctypes.byref(b)))
    return b.value


def token_importance(attn, x, rho: float, important, workspace, importance=None, stream=None):
    """attn: [H][L][L] bf16 bits (int16 tensor), x: [L][d] bf16 bits; writes the
    protected mask (uint8 [L]) and, if given, the importance (float32 [L])."""
    H, L, _ = attn.shape
    d = x.shape[1]
    _check(load().mc_token_importance(_ptr(attn), H, L, _ptr(x), d, ctypes.c_float(rho),
                                      None if importance is None else _ptr(importance), _ptr(important),
                                      _ptr(workspace), workspace.numel() * workspace.element_size(),
                                      _stream(stream)))


def odp_threshold(logits_host):
    """(mu, tau) from calibration logits (a C-contiguous float32 numpy array [T][E])."""
    import numpy as np
    lg = np.ascontiguousarray(logits_host, dtype=np.float32)
    mu, tau = ctypes.c_double(), ctypes.c_double()
    _check(load().mc_odp_threshold(lg.ctypes.data_as(ctypes.c_void_p), lg.shape[0], lg.shape[1],
                                   ctypes.byref(mu), ctypes.byref(tau)))
    return mu.value, tau.value


def pmq_significance(logits_host, k: int):
    """(phi, w) per expert from calibration logits (float32 numpy [T][E])."""
    import numpy as np
    lg = np.ascontiguousarray(logits_host, dtype=np.float32)
    T, E = lg.shape
    phi, w = np.empty(E, np.float64), np.empty(E, np.float64)
    _check(load().mc_pmq_significance(lg.ctypes.data_as(ctypes.c_void_p), T, E, k,
                                      phi.ctypes.data_as(ctypes.c_void_p), w.ctypes.data_as(ctypes.c_void_p)))
    return phi, w


def pmq_allocate(phi, w, eps, total_bits: int, alpha: float = 1.0, beta: float = 1.0, gamma: float = 2.0):
    """Eq. 4 widths: (bits list, objective).  eps: [E][3] errors at 1, 2, 3 bits."""
    import numpy as np
    phi = np.ascontiguousarray(phi, dtype=np.float64)
    w = np.ascontiguousarray(w, dtype=np.float64)
    eps = np.ascontiguousarray(eps, dtype=np.float64)
    E = phi.shape[0]
    bits = np.empty(E, np.int32)
    obj = ctypes.c_double()
    _check(load().mc_pmq_allocate(phi.ctypes.data_as(ctypes.c_void_p), w.ctypes.data_as(ctypes.c_void_p),
                                  eps.ctypes.data_as(ctypes.c_void_p), E, float(alpha), float(beta),
                                  float(gamma), int(total_bits), bits.ctypes.data_as(ctypes.c_void_p),
                                  ctypes.byref(obj)))
    return [int(b) for b in bits], obj.value


def pmq_error_workspace(T: int, E: int, k: int, d: int, ffn: int, group: int) -> int:
    b = ctypes.c_size_t()
    _check(load().mc_pmq_error_workspace(T, E, k, d, ffn, group, ctypes.byref(b)))
    return b.value


def pmq_expert_error(w_gate, w_up, w_down, x, routing: Routing, group: int, workspace, stream=None):
    """eps [E][3] (numpy fp64): the reconstruction error of each expert at 1,
    2 and 3 bits on the calibration batch x [T][d] (bf16 or int16 bits) routed
    by ``routing``; fp32 device weights as for pack()."""
    import numpy as np
    for t in (w_gate, w_up, w_down):
        assert t.dtype == torch.float32 and t.is_contiguous() and t.is_cuda
    assert x.is_contiguous() and x.element_size() == 2 and workspace.is_contiguous()
    E, ffn, d = w_gate.shape
    eps = np.empty((E, 3), np.float64)
    _check(load().mc_pmq_expert_error(_ptr(w_gate), _ptr(w_up), _ptr(w_down), E, d, ffn, int(group), _ptr(x),
                                      ctypes.byref(routing.desc), eps.ctypes.data_as(ctypes.c_void_p),
                                      _ptr(workspace), workspace.numel() * workspace.element_size(),
                                      _stream(stream)))
    return eps


def timing_enable(on: bool = True):
    _check(load().mc_timing_enable(1 if on else 0))


def timing_read(kernel: str):
    """(summed ms, launches) of the events recorded for one kernel."""
    ms, n = ctypes.c_double(), ctypes.c_int()
    _check(load().mc_timing_read(kernel.encode(), ctypes.byref(ms), ctypes.byref(n)))
    return ms.value, n.value
