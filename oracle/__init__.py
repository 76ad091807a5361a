"""CPU oracle of the Mixture Compressor expert path -- TEST INFRASTRUCTURE.

Only ``tests/``, ``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of
``bench.py`` may import this package.  The product library never calls it and
shares no code with it: the kernels and the C functions in ``mc_oracle.c``
implement the same definitions independently.

What it computes (Mixture Compressor for MoE LLMs, ICLR 2025):

* ``quantize``      -- Sec. 3.1 uniform asymmetric group quantizer (fp16 scale
  and zero, codes in [0, 2^b - 1], nearest level decided exactly);
* ``quantize_sign`` -- appendix A.2 sign binarization of 1-bit experts, in
  the same group format (scale 2 mean|W|, zero 1/2);
* ``layout_pack`` / ``layout_unpack`` / ``pack_sz`` / ``unpack_sz`` -- the
  packed storage format, element by element from its index function;
* ``dequant_f16`` / ``dequant_exact`` -- the dequantized value s*(q - z);
* ``gptq_hessian`` / ``gptq_quantize`` -- the GPTQ quantizer the paper uses
  (Sec. 3.1; H = 2 X^T X, columns quantized in order, each column's error
  compensated on the columns after it through the upper Cholesky factor of
  H^-1), with the group parameters of the Sec. 3.1 quantizer;
* ``router_logits`` -- the router's linear layer x W_r^T whose top-k Eq. 1
  takes, each logit the exact sum rounded once to fp32;
* ``route``         -- Eq. 1 top-k, Eq. 5 pruning, Sec. 3.3.2 protection and
  the per-expert token lists;
* ``moe_forward``   -- Eq. 1 over SwiGLU experts on exact dequantized weights;
* ``rms_norm`` / ``moe_stack`` -- layers of Eq. 1, each behind an RMSNorm,
  joined by residual connections, the stream rounded to bfloat16 after each
  layer;
* ``token_importance`` -- Eq. 6 importance from causal attention probabilities
  and the protected set (the top floor(rho*L + 1/2) tokens);
* ``median_ratio``  -- the pruning threshold mu as the median of w1/w0;
* ``pmq_significance`` / ``pmq_allocate`` -- Sec. 3.2: expert access
  frequency and mean routing weight, and the Eq. 4 width allocation;
* ``pmq_expert_error`` -- Sec. 3.2.2: the F-norm change of one MoE layer's
  output when only expert e is quantized at b bits (the errors Eq. 4 takes),
  with ``dense_expert_forward`` the unquantized SwiGLU expert.

Everything floating point is fp64 except operations whose precision the
definition fixes (fp32 scale/zero arithmetic, the fp32 k = 2 logit gap).
Parity status of each function is recorded in ``PINS`` below.
"""
from __future__ import annotations

import ctypes
import math
import os
import subprocess
import threading

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "mc_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lock = threading.Lock()
_lib = None

# Every function is pinned by tests that do not re-use its own code
# (see tests/test_oracle_pins.py); none is "parity unpinned".
PINS = {
    "quantize": "Fraction brute force over all codes; level bound; range endpoints",
    "quantize_sign": "Eq. 7-9: 2 code - 1 = sign(W) with sign(0) = +1; dequantized = +-mean|W| "
                     "to fp16 rounding; Eq. 10 add/subtract form of the product",
    "layout_pack": "round trip, word-count closed form, hand-built words",
    "dequant_f16": "Fraction value rounded by numpy float16 (library RNE)",
    "gptq_factor": "U^T U H = I; upper triangular with positive diagonal; dead inputs; damping scale",
    "gptq_quantize": "H = c I reduces to RTN bit for bit; two-column closed form (w1 + rho (w0 - q0)); "
                     "loss identity d H d^T = sum e^2; error below RTN's on correlated inputs; dead inputs",
    "codes_for": "equals the quantizer's own codes when the parameters come from the same values",
    "router_logits": "Fraction sums rounded to the nearest fp32 by exact distance; hand cases "
                     "with cancellation, fp32 ties and double-rounding traps; fp64 matmul within 1 ulp",
    "route": "naive stable sort; tau=0 and protected no-op; k=2 gap == ratio rule",
    "moe_forward": "E=1,k=1 equals numpy SwiGLU; tau=0 all-protected dense top-k; linearity",
    "rms_norm": "torch.nn.functional.rms_norm in float64; scale invariance; unit mean square",
    "moe_stack": "numpy residual SwiGLU stack at E=1,k=1; zero experts are the identity; "
                 "tokens are independent (a subset matches the full run)",
    "token_importance": "diagonal / first-token closed forms; hand example; head linearity; "
                        "brute-force selection; upper triangle ignored",
    "median_ratio": "statistics.median of exp(l1 - l0) over a naive sort",
    "pmq_significance": "hand example (golden); sum phi = k and sum w = 1; tie order",
    "pmq_allocate": "hand-enumerated example (golden); enumeration of every width vector; "
                    "constraints; significance ordering",
    "dense_expert_forward": "one hand-computed token (closed-form silu); linearity of the down projection",
    "pmq_expert_error": "the definition taken literally (two whole-layer outputs, one with only expert e "
                        "quantized); zero for an expert no token keeps; zero at 1 bit for weights on "
                        "the 1-bit grid; equal to the per-token brute-force sum",
}


def build(force: bool = False) -> str:
    """Compile ``liboracle.so`` with gcc (plain C, no fast-math, no contraction)."""
    with _lock:
        if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
            tmp = _LIB + ".tmp%d" % os.getpid()
            subprocess.check_call([
                "gcc", "-O2", "-std=c99", "-ffp-contract=off", "-fno-fast-math",
                "-fopenmp", "-fPIC", "-shared", "-o", tmp, _SRC, "-lm"])
            os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        build()
        lib = ctypes.CDLL(_LIB)
        P = ctypes.c_void_p
        I = ctypes.c_int
        lib.orc_f16_to_double.restype = ctypes.c_double
        lib.orc_f16_to_double.argtypes = [ctypes.c_uint16]
        for name in ("orc_f16_from_double", "orc_f16_from_double_sat", "orc_bf16_from_double"):
            getattr(lib, name).restype = ctypes.c_uint16
            getattr(lib, name).argtypes = [ctypes.c_double]
        lib.orc_bf16_to_double.restype = ctypes.c_double
        lib.orc_bf16_to_double.argtypes = [ctypes.c_uint16]
        lib.orc_quantize_group.restype = I
        lib.orc_quantize_group.argtypes = [P, I, I, P, P, P]
        lib.orc_quantize_matrix.restype = I
        lib.orc_quantize_matrix.argtypes = [P, I, I, I, I, P, P, P]
        lib.orc_dequant.restype = ctypes.c_double
        lib.orc_dequant.argtypes = [ctypes.c_uint16, ctypes.c_uint16, I]
        lib.orc_dequant_matrix_f16.restype = None
        lib.orc_dequant_matrix_f16.argtypes = [P, P, P, I, I, I, P]
        lib.orc_layout_pack.restype = I
        lib.orc_layout_pack.argtypes = [P, I, I, I, P]
        lib.orc_layout_unpack.restype = I
        lib.orc_layout_unpack.argtypes = [P, I, I, I, P]
        lib.orc_layout_pack_sz.restype = I
        lib.orc_layout_pack_sz.argtypes = [P, P, I, I, I, P]
        lib.orc_layout_unpack_sz.restype = I
        lib.orc_layout_unpack_sz.argtypes = [P, I, I, I, P, P]
        lib.orc_route.restype = I
        lib.orc_route.argtypes = [P, P, I, I, I, ctypes.c_double, ctypes.c_float,
                                  P, P, P, P, P, P, P, P, P, P]
        lib.orc_expert_forward.restype = I
        lib.orc_token_importance.argtypes = [P, I, I, P, I, I, P, P]
        lib.orc_token_importance.restype = I
        lib.orc_median_ratio.argtypes = [P, I, I]
        lib.orc_median_ratio.restype = ctypes.c_double
        lib.orc_expert_forward.argtypes = [P, I, I, I, I, P, P, P, P, P, P, P, P, P, P, I, P, P]
        _lib = lib
    return _lib


def _p(a: np.ndarray):
    assert a.flags["C_CONTIGUOUS"]
    return a.ctypes.data_as(ctypes.c_void_p)


# ---------------------------------------------------------------- formats ---

def f16_to_float(h: int) -> float:
    return _load().orc_f16_to_double(int(h))


def f16_round(v: float, saturate: bool = False) -> int:
    lib = _load()
    return int(lib.orc_f16_from_double_sat(v) if saturate else lib.orc_f16_from_double(v))


def bf16_round(v: float) -> int:
    return int(_load().orc_bf16_from_double(float(v)))


def bf16_round_array(a: np.ndarray) -> np.ndarray:
    """Round-to-nearest-even bfloat16 bits of each fp64 value (element loop in C)."""
    lib = _load()
    flat = np.ascontiguousarray(a, dtype=np.float64).ravel()
    out = np.empty(flat.shape, dtype=np.uint16)
    for i, v in enumerate(flat):
        out[i] = lib.orc_bf16_from_double(float(v))
    return out.reshape(np.shape(a))


def bf16_to_float64(h: np.ndarray) -> np.ndarray:
    """Exact widening of bfloat16 bit patterns."""
    h = np.asarray(h, dtype=np.uint16)
    return (h.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


# -------------------------------------------------------------- quantizer ---

def quantize_group(w: np.ndarray, bits: int):
    """Sec. 3.1 quantizer on one group: returns (s16 bits, z16 bits, codes)."""
    w = np.ascontiguousarray(w, dtype=np.float32)
    s = np.zeros(1, np.uint16)
    z = np.zeros(1, np.uint16)
    q = np.zeros(w.size, np.uint8)
    if _load().orc_quantize_group(_p(w), w.size, bits, _p(s), _p(z), _p(q)):
        raise ValueError("bad quantize_group arguments")
    return int(s[0]), int(z[0]), q


def quantize(W: np.ndarray, bits: int, G: int):
    """Row-major W[R][K] -> (codes uint8 [R][K], s16 [R][K/G], z16 [R][K/G])."""
    W = np.ascontiguousarray(W, dtype=np.float32)
    R, K = W.shape
    q = np.empty((R, K), np.uint8)
    s = np.empty((R, K // G), np.uint16)
    z = np.empty((R, K // G), np.uint16)
    if _load().orc_quantize_matrix(_p(W), R, K, G, bits, _p(q), _p(s), _p(z)):
        raise ValueError("bad quantize arguments")
    return q, s, z


def dequant_exact(q: np.ndarray, s: np.ndarray, z: np.ndarray, G: int) -> np.ndarray:
    """s*(q - z) in fp64 (exact: see the quantizer comment in mc_oracle.c)."""
    sf = s.view(np.float16).astype(np.float64)
    zf = z.view(np.float16).astype(np.float64)
    sf = np.repeat(sf, G, axis=1)
    zf = np.repeat(zf, G, axis=1)
    return sf * (q.astype(np.float64) - zf)


def dequant_f16(q: np.ndarray, s: np.ndarray, z: np.ndarray, G: int) -> np.ndarray:
    """fp16 bits of the single RNE rounding of s*(q - z)."""
    R, K = q.shape
    out = np.empty((R, K), np.uint16)
    _load().orc_dequant_matrix_f16(_p(np.ascontiguousarray(q)), _p(np.ascontiguousarray(s)),
                                   _p(np.ascontiguousarray(z)), R, K, G, _p(out))
    return out


# ----------------------------------------------------------------- layout ---

def layout_pack(q: np.ndarray, bits: int) -> np.ndarray:
    q = np.ascontiguousarray(q, dtype=np.uint8)
    R, K = q.shape
    words = np.empty(R * K * bits // 32, np.uint32)
    if _load().orc_layout_pack(_p(q), R, K, bits, _p(words)):
        raise ValueError("shape not packable")
    return words


def layout_unpack(words: np.ndarray, R: int, K: int, bits: int) -> np.ndarray:
    words = np.ascontiguousarray(words, dtype=np.uint32)
    assert words.size == R * K * bits // 32
    q = np.empty((R, K), np.uint8)
    if _load().orc_layout_unpack(_p(words), R, K, bits, _p(q)):
        raise ValueError("shape not packable")
    return q


def pack_sz(s: np.ndarray, z: np.ndarray, G: int) -> np.ndarray:
    s = np.ascontiguousarray(s, dtype=np.uint16)
    z = np.ascontiguousarray(z, dtype=np.uint16)
    R, ng = s.shape
    out = np.empty(R * ng, np.uint32)
    if _load().orc_layout_pack_sz(_p(s), _p(z), R, ng * G, G, _p(out)):
        raise ValueError("shape not packable")
    return out


def unpack_sz(sz: np.ndarray, R: int, K: int, G: int):
    sz = np.ascontiguousarray(sz, dtype=np.uint32)
    s = np.empty((R, K // G), np.uint16)
    z = np.empty((R, K // G), np.uint16)
    if _load().orc_layout_unpack_sz(_p(sz), R, K, G, _p(s), _p(z)):
        raise ValueError("shape not packable")
    return s, z


def layer_offsets(E: int, d: int, ffn: int, bits, G: int):
    """Word and scale/zero-word offsets of (expert, matrix) inside a layer:
    experts in order, each holding gate [ffn][d], up [ffn][d], down [d][ffn]."""
    words, szs = {}, {}
    wo = so = 0
    for e in range(E):
        for m in range(3):
            words[(e, m)] = wo
            szs[(e, m)] = so
            wo += d * ffn * int(bits[e]) // 32
            so += d * ffn // G
    return words, szs, wo, so


def quantize_sign(W: np.ndarray, G: int):
    """Appendix A.2 (Eq. 7-9) in the group format: B = sign(W) with sign(0) =
    +1, stored as B~ = (B + 1)/2 (code 1 where w >= 0, -0 included); one scale
    for the matrix, s = ||W||_1 / (rows * cols), kept in every group as
    fp16(2 s) (saturating) with zero 1/2, so that s16 * (code - 1/2) =
    +-s16 / 2.  ||W||_1 is summed exactly (math.fsum) and rounded once."""
    W = np.asarray(W, dtype=np.float32)
    R, K = W.shape
    q = (W >= 0).astype(np.uint8)
    l1 = math.fsum(float(v) for v in np.abs(W).ravel())
    s2 = 2.0 * (l1 / (R * K))
    s16 = f16_round(min(s2, 65504.0))
    s = np.full((R, K // G), s16, np.uint16)
    z = np.full((R, K // G), 0x3800, np.uint16)          # fp16 0.5
    return q, s, z


def pack_layer(mats, bits, G: int, methods=None):
    """mats[e] = (gate [ffn][d], up [ffn][d], down [d][ffn]) fp32; methods[e]
    = 0 (min-max RTN, ``quantize``) or 1 (sign binarization, 1-bit experts).
    Returns (words uint32, sz uint32, logical) with logical[e][m] = (q, s, z)."""
    E = len(mats)
    ffn, d = mats[0][0].shape
    wofs, sofs, nw, ns = layer_offsets(E, d, ffn, bits, G)
    words = np.zeros(nw, np.uint32)
    sz = np.zeros(ns, np.uint32)
    logical = []
    for e in range(E):
        per = []
        for m in range(3):
            if methods is not None and methods[e] == 1:
                assert int(bits[e]) == 1
                q, s, z = quantize_sign(mats[e][m], G)
            else:
                q, s, z = quantize(mats[e][m], int(bits[e]), G)
            w = layout_pack(q, int(bits[e]))
            words[wofs[(e, m)]: wofs[(e, m)] + w.size] = w
            p = pack_sz(s, z, G)
            sz[sofs[(e, m)]: sofs[(e, m)] + p.size] = p
            per.append((q, s, z))
        logical.append(per)
    return words, sz, logical


# ---------------------------------------------------------------- routing ---

def codes_for(w32: np.ndarray, s16: np.ndarray, z16: np.ndarray, bits: int) -> np.ndarray:
    """Nearest level code of each fp32 value w under fp16 scale/zero bits
    (one per value): the number of level midpoints s*(j + 1/2 - z) below w,
    the even neighbour when w is exactly on a midpoint (midpoints are exact
    in fp64)."""
    L = (1 << bits) - 1
    w = np.asarray(w32, dtype=np.float32).astype(np.float64)
    s = np.asarray(s16, np.uint16).view(np.float16).astype(np.float64)
    z = np.asarray(z16, np.uint16).view(np.float16).astype(np.float64)
    below = np.zeros(w.shape, np.int64)
    for j in range(L):
        below += (s * ((j + 0.5) - z) < w)
    on_mid = (below < L) & (below % 2 == 1) & (s * ((below + 0.5) - z) == w)
    return (below + on_mid).astype(np.uint8)


def gptq_hessian(x_bits: np.ndarray) -> np.ndarray:
    """H = 2 X^T X (fp64) from calibration inputs X [N][K] (bf16 bits): the
    Hessian in W of the layer-wise error ||W X^T - Q X^T||^2 (Sec. 3.1)."""
    X = bf16_to_float64(x_bits)
    return 2.0 * (X.T @ X)


def _f32_margin(w64: np.ndarray) -> np.ndarray:
    """Relative distance of each fp64 value to the nearest fp32 rounding
    boundary (how far it is from rounding to another fp32)."""
    f = w64.astype(np.float32)
    up = np.nextafter(f, np.float32(np.inf)).astype(np.float64)
    dn = np.nextafter(f, np.float32(-np.inf)).astype(np.float64)
    fd = f.astype(np.float64)
    dist = np.minimum(np.abs(w64 - (fd + up) / 2), np.abs(w64 - (fd + dn) / 2))
    return dist / np.maximum(np.abs(w64), 1e-300)


def gptq_factor(H: np.ndarray, damp: float = 0.01):
    """The factor GPTQ quantizes with, from the Hessian H [K][K] (fp64):
    inputs with H_kk = 0 are dead (H_kk := 1; their weights are zeroed);
    H += damp * mean(diag H) * I; U = the upper-triangular Cholesky factor of
    H^-1 (H^-1 = U^T U).  Returns (U [K][K] fp64, dead [K] uint8)."""
    H = np.array(H, dtype=np.float64, copy=True)
    K = H.shape[0]
    dead = np.diag(H) == 0.0
    H[dead, dead] = 1.0
    H[np.diag_indices(K)] += damp * np.mean(np.diag(H))
    U = np.linalg.cholesky(np.linalg.inv(H)).T
    return np.triu(U), dead.astype(np.uint8)


def gptq_quantize_u(W: np.ndarray, U: np.ndarray, dead: np.ndarray, bits: int, G: int):
    """GPTQ on one matrix W [R][K] (rows = outputs, K = inputs) with the
    factor U of ``gptq_factor``, in fp64.  Dead inputs get weight 0; then for
    k = 0 .. K-1 (columns in order):
      at a group start, s and z come from the Sec. 3.1 quantizer on the fp32
      rounding of the group's current (already compensated) values;
      q_k = nearest level of fp32(w_k);  e_k = (w_k - s (q_k - z)) / U_kk;
      w_j -= e_k U_kj for every j > k.
    Returns (q [R][K] uint8, s16 [R][K/G], z16 [R][K/G], loss [R] = sum e_k^2
    / 2, margin [R]): margin is the smallest, over the row's decisions, of the
    relative distance of w_k to an fp32 rounding boundary and of fp32(w_k) to a
    level midpoint (in units of s); a row with a tiny margin can round the
    other way under a different fp64 summation order."""
    W = np.asarray(W, dtype=np.float32)
    R, K = W.shape
    Wk = W.astype(np.float64)
    Wk[:, np.asarray(dead, bool)] = 0.0
    L = (1 << bits) - 1
    q = np.zeros((R, K), np.uint8)
    s = np.zeros((R, K // G), np.uint16)
    z = np.zeros((R, K // G), np.uint16)
    loss = np.zeros(R)
    margin = np.full(R, np.inf)
    for k in range(K):
        g = k // G
        if k % G == 0:
            _, sg, zg = quantize(Wk[:, k:k + G].astype(np.float32), bits, G)
            s[:, g], z[:, g] = sg[:, 0], zg[:, 0]
            sf = s[:, g].view(np.float16).astype(np.float64)
            zf = z[:, g].view(np.float16).astype(np.float64)
        w64 = Wk[:, k]
        w32 = w64.astype(np.float32)
        qk = codes_for(w32, s[:, g], z[:, g], bits)
        q[:, k] = qk
        mids = sf[:, None] * ((np.arange(L) + 0.5)[None, :] - zf[:, None])
        dmid = np.abs(w32.astype(np.float64)[:, None] - mids).min(axis=1) / sf
        margin = np.minimum(margin, np.minimum(_f32_margin(w64), dmid))
        err = (w64 - sf * (qk.astype(np.float64) - zf)) / U[k, k]
        Wk[:, k + 1:] -= np.outer(err, U[k, k + 1:])
        loss += err * err / 2.0
    return q, s, z, loss, margin


def gptq_quantize(W: np.ndarray, H: np.ndarray, bits: int, G: int, damp: float = 0.01):
    """GPTQ from the Hessian: ``gptq_quantize_u`` with ``gptq_factor(H, damp)``."""
    U, dead = gptq_factor(H, damp)
    return gptq_quantize_u(W, U, dead, bits, G)


def _round_f32(terms) -> float:
    """The fp32 nearest to the exact sum of the fp64 values ``terms`` (ties to
    even); a zero sum is +0.  math.fsum gives s, the fp64 nearest to the sum,
    and the fp64 nearest to the remainder (so its sign); the cast of s to fp32
    is then correct except when s falls exactly halfway between two fp32
    values, where the remainder's sign decides."""
    s = math.fsum(terms)
    if s == 0.0:
        return 0.0
    r = math.fsum(list(terms) + [-s])
    f = np.float32(s)
    if float(f) == s or r == 0.0:
        return float(f)
    lo = np.nextafter(f, np.float32(-np.inf)) if float(f) > s else f
    hi = np.nextafter(lo, np.float32(np.inf))
    if (float(lo) + float(hi)) / 2.0 != s:        # not a midpoint: the cast is right
        return float(f)
    return float(hi) if r > 0.0 else float(lo)


def router_logits(x_bits: np.ndarray, w_bits: np.ndarray, tokens=None) -> np.ndarray:
    """Router scores whose top-k Eq. 1 takes: logits[t][e] = sum_k x[t][k] *
    W_r[e][k] for bf16 x [T][d] and W_r [E][d] (bit patterns), each the exact
    sum rounded once to fp32 (bf16 products are exact in fp64).  ``tokens``
    restricts the rows computed (others stay 0)."""
    x = bf16_to_float64(x_bits)
    w = bf16_to_float64(w_bits)
    T, E = x.shape[0], w.shape[0]
    out = np.zeros((T, E), dtype=np.float32)
    for t in (range(T) if tokens is None else tokens):
        for e in range(E):
            out[t, e] = _round_f32((x[t] * w[e]).tolist())
    return out


def prune_delta(tau: float) -> float:
    """fp32 threshold on the logit gap l_0 - l_1 equivalent to p_1 < tau at k = 2:
    p_1 = 1 / (1 + exp(l_0 - l_1)) < tau  <=>  l_0 - l_1 > ln((1 - tau) / tau)."""
    if tau <= 0.0:
        return math.inf
    if tau >= 1.0:
        return -math.inf
    return float(np.float32(math.log((1.0 - tau) / tau)))


def route(logits: np.ndarray, important, k: int, tau: float):
    logits = np.ascontiguousarray(logits, dtype=np.float32)
    T, E = logits.shape
    imp = None if important is None else np.ascontiguousarray(important, dtype=np.uint8)
    out = dict(
        topk_idx=np.empty((T, k), np.int32), topk_w=np.empty((T, k), np.float64),
        kept=np.empty((T, k), np.uint8), counts=np.empty(E, np.int32),
        offsets=np.empty(E + 1, np.int32), pair_token=np.full(T * k, -1, np.int32),
        pair_rank=np.full(T * k, -1, np.int32), pair_w=np.zeros(T * k, np.float64),
        pair_pos=np.empty((T, k), np.int32), n_pruned=np.zeros(1, np.int32))
    rc = _load().orc_route(
        _p(logits), None if imp is None else _p(imp), T, E, k, float(tau),
        ctypes.c_float(prune_delta(tau)),
        _p(out["topk_idx"]), _p(out["topk_w"]), _p(out["kept"]), _p(out["counts"]),
        _p(out["offsets"]), _p(out["pair_token"]), _p(out["pair_rank"]), _p(out["pair_w"]),
        _p(out["pair_pos"]), _p(out["n_pruned"]))
    if rc:
        raise ValueError("bad route arguments")
    out["n_pruned"] = int(out["n_pruned"][0])
    return out


# ---------------------------------------------------------------- forward ---

def expert_forward(X: np.ndarray, logical_e, G: int, rows=None):
    """One SwiGLU expert on token rows X [nt][d] (fp64).  Returns (H [nt][ffn],
    Y [nt][len(rows) or d])."""
    X = np.ascontiguousarray(X, dtype=np.float64)
    nt, d = X.shape
    (qg, sg, zg), (qu, su, zu), (qd, sd, zd) = logical_e
    ffn = qg.shape[0]
    H = np.empty((nt, ffn), np.float64)
    if rows is None:
        rows_a, nr = None, d
    else:
        rows_a = np.ascontiguousarray(rows, dtype=np.int32)
        nr = rows_a.size
    Y = np.empty((nt, nr), np.float64)
    c = np.ascontiguousarray
    rc = _load().orc_expert_forward(
        _p(X), nt, d, ffn, G, _p(c(qg)), _p(c(sg)), _p(c(zg)), _p(c(qu)), _p(c(su)), _p(c(zu)),
        _p(c(qd)), _p(c(sd)), _p(c(zd)), None if rows_a is None else _p(rows_a), nr, _p(H), _p(Y))
    if rc:
        raise ValueError("bad expert_forward arguments")
    return H, Y


def moe_forward(x_bf16: np.ndarray, routing, logical, G: int, rows=None, tokens=None) -> np.ndarray:
    """Eq. 1: y_t = sum over kept ranks of w_r * E_{e_r}(x_t), fp64.
    ``rows`` restricts the output columns, ``tokens`` the output tokens."""
    X = bf16_to_float64(x_bf16)
    T, d = X.shape
    toks = np.arange(T) if tokens is None else np.asarray(tokens)
    nr = d if rows is None else len(rows)
    Y = np.zeros((len(toks), nr), np.float64)
    tpos = {int(t): i for i, t in enumerate(toks)}
    E = len(logical)
    k = routing["topk_idx"].shape[1]
    for e in range(E):
        sel = [(int(t), r) for t in toks for r in range(k)
               if routing["topk_idx"][t, r] == e and routing["kept"][t, r]]
        if not sel:
            continue
        Xe = X[[t for t, _ in sel]]
        _, Ye = expert_forward(Xe, logical[e], G, rows)
        for i, (t, r) in enumerate(sel):
            Y[tpos[t]] += routing["topk_w"][t, r] * Ye[i]
    return Y


RMS_EPS = 1e-5


def rms_norm(h_bf16: np.ndarray, eps: float = RMS_EPS) -> np.ndarray:
    """Per row: bf16(h / sqrt(mean(h^2) + eps)) (unit gain), the value formed
    in fp64 and rounded once; returns bf16 bits."""
    H = bf16_to_float64(np.asarray(h_bf16, dtype=np.uint16))
    r = 1.0 / np.sqrt((H * H).mean(axis=1, keepdims=True) + eps)
    return bf16_round_array(H * r)


def moe_stack(x_bf16: np.ndarray, layers, G: int, tokens=None):
    """Residual stack of MoE layers, each behind its RMSNorm:
    h_0 = x, xn_l = rms_norm(h_l), h_{l+1} = RNE_bf16(h_l + y_l) with y_l =
    Eq. 1 of layer l on xn_l (fp64, exact dequantized weights).
    ``layers``: list of (routing, logical) with routing from ``route``.
    ``tokens`` restricts the computation to those tokens (each token's path
    depends only on its own row).  Returns the list of bf16 bit arrays
    h_1 .. h_n, rows in the order of ``tokens`` (all tokens by default)."""
    x_bf16 = np.asarray(x_bf16, dtype=np.uint16)
    T = x_bf16.shape[0]
    toks = np.arange(T) if tokens is None else np.asarray(tokens)
    H = x_bf16.copy()
    outs = []
    for routing, logical in layers:
        XN = H.copy()
        XN[toks] = rms_norm(H[toks])
        Y = moe_forward(XN, routing, logical, G, tokens=toks)
        H[toks] = bf16_round_array(bf16_to_float64(H[toks]) + Y)
        outs.append(H[toks].copy())
    return outs


# -------------------------------------------------------------------- PMQ ---

def pmq_significance(logits: np.ndarray, k: int):
    """Sec. 3.2.1: over N calibration tokens, phi_e = n_e / N with n_e the
    tokens whose top-k contains e, and w_e = (sum of e's routing weights) / N,
    the routing weights being the softmax over the selected k (Eq. 1
    convention of ``route``).  Plain loops in fp64."""
    T, E = logits.shape
    n = [0.0] * E
    s = [0.0] * E
    for t in range(T):
        row = [float(v) for v in logits[t]]
        order = sorted(range(E), key=lambda e: (-row[e], e))[:k]
        ex = [math.exp(row[e] - row[order[0]]) for e in order]
        tot = 0.0
        for v in ex:
            tot += v
        for e, v in zip(order, ex):
            n[e] += 1.0
            s[e] += v / tot
    return np.array([v / T for v in n]), np.array([v / T for v in s])


def _pmq_terms(phi, w, eps, alpha, beta, gamma):
    return [[(float(phi[i]) ** alpha) * (float(w[i]) ** beta) * (float(eps[i][b]) ** gamma)
             for b in range(3)] for i in range(len(phi))]


def _pmq_feasible(bits, total):
    return sum(bits) == total and 3 in bits and 2 in bits


def pmq_allocate_bruteforce(phi, w, eps, total_bits: int, alpha=1.0, beta=1.0, gamma=2.0):
    """Eq. 4 by enumeration of every width vector in lexicographic order (for
    small E): minimise sum_i phi_i^alpha w_i^beta eps_{i,b_i}^gamma (terms
    added in expert order) subject to sum b_i = total_bits, some b_i = 3 and
    some b_i = 2; the first minimum met (the lexicographically smallest) wins.
    Returns (bits, objective) or None when infeasible."""
    import itertools
    term = _pmq_terms(phi, w, eps, alpha, beta, gamma)
    best = None
    for bits in itertools.product((1, 2, 3), repeat=len(phi)):
        if not _pmq_feasible(bits, total_bits):
            continue
        c = 0.0
        for i, b in enumerate(bits):
            c += term[i][b - 1]
        if best is None or c < best[1]:
            best = (list(bits), c)
    return best


def pmq_allocate(phi, w, eps, total_bits: int, alpha=1.0, beta=1.0, gamma=2.0):
    """Eq. 4 for any E: dynamic programme over experts in order; a state is
    (bits used, some expert at 2, some at 3) and keeps its cheapest prefix
    (cost summed in expert order; equal costs keep the lexicographically
    smaller prefix).  Same result as the enumeration."""
    term = _pmq_terms(phi, w, eps, alpha, beta, gamma)
    states = {(0, False, False): (0.0, [])}
    for i in range(len(phi)):
        nxt = {}
        for (s, h2, h3), (c, pre) in sorted(states.items()):
            for b in (1, 2, 3):
                key = (s + b, h2 or b == 2, h3 or b == 3)
                cand = (c + term[i][b - 1], pre + [b])
                if key not in nxt or cand[0] < nxt[key][0] or (cand[0] == nxt[key][0] and cand[1] < nxt[key][1]):
                    nxt[key] = cand
        states = nxt
    got = states.get((total_bits, True, True))
    return None if got is None else (got[1], got[0])


# ------------------------------------------------------------- importance ---

def dense_expert_forward(X: np.ndarray, Wg: np.ndarray, Wu: np.ndarray, Wd: np.ndarray) -> np.ndarray:
    """The SwiGLU expert with unquantized weights, fp64: rows of X [n][d] ->
    Wd (silu(Wg x) * (Wu x)); Wg, Wu [ffn][d], Wd [d][ffn]."""
    X = np.asarray(X, dtype=np.float64)
    g = X @ np.asarray(Wg, dtype=np.float64).T
    u = X @ np.asarray(Wu, dtype=np.float64).T
    h = g / (1.0 + np.exp(-g)) * u
    return h @ np.asarray(Wd, dtype=np.float64).T


def pmq_expert_error(Wg, Wu, Wd, x_bf16: np.ndarray, routing, G: int) -> np.ndarray:
    """Sec. 3.2.2: eps[e][b-1] = ||F(theta) - F(theta[e -> Q(e, b)])||_F for
    b = 1, 2, 3, F the MoE layer output (Eq. 1) over the batch, theta the
    fp32 weights Wg, Wu [E][ffn][d], Wd [E][d][ffn], Q the Sec. 3.1 quantizer
    (``quantize``) at b bits, group size G.  Only the tokens that keep e see
    the change, by w_r (E_e^(b)(x_t) - E_e(x_t)) each, so eps[e][b-1]^2 sums
    the squared norms of those terms; the quantized expert runs on its exact
    dequantized weights (``expert_forward``)."""
    X = bf16_to_float64(x_bf16)
    E = len(Wg)
    k = routing["topk_idx"].shape[1]
    T = X.shape[0]
    eps = np.zeros((E, 3), np.float64)
    for e in range(E):
        sel = [(t, r) for t in range(T) for r in range(k)
               if routing["topk_idx"][t, r] == e and routing["kept"][t, r]]
        if not sel:
            continue
        Xe = X[[t for t, _ in sel]]
        w = np.array([routing["topk_w"][t, r] for t, r in sel], np.float64)
        Y = dense_expert_forward(Xe, Wg[e], Wu[e], Wd[e])
        for b in (1, 2, 3):
            logical_e = [quantize(np.asarray(W[e], np.float32), b, G) for W in (Wg, Wu, Wd)]
            _, Yq = expert_forward(Xe, logical_e, G)
            eps[e, b - 1] = math.sqrt(float((((Yq - Y) * w[:, None]) ** 2).sum()))
    return eps


def protect_count(L: int, rho: float) -> int:
    """Tokens protected out of L at fraction rho: floor(rho * L + 1/2)."""
    return int(math.floor(rho * L + 0.5))


def token_importance(attn_bits: np.ndarray, x_bits: np.ndarray, rho: float):
    """Eq. 6 from attention probabilities attn [H][L][L] (bf16 bits, query-major,
    causal) and tokens x [L][d] (bf16 bits).  Returns (I [L] fp64, mask [L] uint8)."""
    attn_bits = np.ascontiguousarray(attn_bits, dtype=np.uint16)
    x_bits = np.ascontiguousarray(x_bits, dtype=np.uint16)
    H, L, L2 = attn_bits.shape
    assert L == L2 and x_bits.shape[0] == L
    d = x_bits.shape[1]
    I = np.empty(L, np.float64)
    mask = np.empty(L, np.uint8)
    rc = _load().orc_token_importance(_p(attn_bits), H, L, _p(x_bits), d, protect_count(L, rho),
                                      _p(I), _p(mask))
    if rc:
        raise ValueError("bad token_importance arguments")
    return I, mask


def median_ratio(logits: np.ndarray) -> float:
    """mu = median over tokens of w1/w0 of the top-2 experts (Sec. 3.3.1)."""
    logits = np.ascontiguousarray(logits, dtype=np.float32)
    T, E = logits.shape
    mu = _load().orc_median_ratio(_p(logits), T, E)
    if mu < 0:
        raise ValueError("bad median_ratio arguments")
    return mu
