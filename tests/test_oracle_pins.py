"""Pins of the CPU oracle against what the paper and the mathematics fix.

None of these tests re-types an oracle formula: each compares the oracle with
an independent route (exact rational brute force, a library routine, a
hand-derived fixture, a closed form or an invariant), chosen so that a dropped
term, a wrong sign, index or tie rule, or a transposed operand fails one.
"""
import math
import os
from fractions import Fraction

import numpy as np
import pytest
import scipy.special

import oracle
import synthetic

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _lines(name):
    with open(os.path.join(GOLD, name)) as f:
        for line in f:
            line = line.strip()
            if line and not line.startswith("#"):
                yield [p.strip() for p in line.split("|")]


def f16val(bits):
    return float(np.array([bits], np.uint16).view(np.float16)[0])


# --------------------------------------------------------------- formats ---

def test_f16_rounding_matches_numpy():
    """RNE to fp16 (Sec. 3.1 stores scale and zero in 16 bits) vs numpy's float16 cast."""
    g = np.random.default_rng(1)
    vals = np.concatenate([
        g.standard_normal(4000) * 10.0 ** g.integers(-9, 5, 4000),
        np.array([65504.0, 65519.99, 65520.0, 65536.0, 2.0 ** -24, 2.0 ** -25, 3 * 2.0 ** -26,
                  2.0 ** -14, 2.0 ** -14 - 2.0 ** -25, 1.0 + 2.0 ** -11, 1.0 + 3 * 2.0 ** -11,
                  0.0, -0.0, -1.5, 2049.0, 2051.0]),
    ])
    for v in vals:
        with np.errstate(over="ignore"):
            want = int(np.array([v], np.float64).astype(np.float16).view(np.uint16)[0])
        assert oracle.f16_round(float(v)) == want, v


def test_f16_saturating():
    assert oracle.f16_round(1e6, saturate=True) == 0x7BFF
    assert oracle.f16_round(-1e6, saturate=True) == 0xFBFF
    assert oracle.f16_round(65519.0, saturate=True) == 0x7BFF
    assert oracle.f16_round(1e6) == 0x7C00


def test_bf16_rounding_matches_torch():
    torch = pytest.importorskip("torch")
    g = np.random.default_rng(2)
    v = (g.standard_normal(5000) * 10.0 ** g.integers(-30, 30, 5000)).astype(np.float32)
    want = torch.from_numpy(v).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    got = oracle.bf16_round_array(v.astype(np.float64))
    np.testing.assert_array_equal(got, want)


# -------------------------------------------------------------- quantizer ---

def _brute_codes(w, s16, z16, bits):
    """argmin_j |w - s*(j - z)| over all 2^b codes in exact rationals, ties -> even j."""
    s = Fraction(f16val(s16))
    z = Fraction(f16val(z16))
    out = []
    for wi in w:
        wf = Fraction(float(wi))
        best = None
        for j in range(2 ** bits):
            dist = abs(wf - s * (j - z))
            if best is None or dist < best[0] or (dist == best[0] and j % 2 == 0):
                best = (dist, j)
        out.append(best[1])
    return out


@pytest.mark.parametrize("bits", [1, 2, 3])
def test_quantizer_codes_are_exact_nearest_levels(bits):
    g = np.random.default_rng(10 + bits)
    for trial in range(40):
        G = 32
        w = (g.standard_normal(G) * 0.02 * (1 + trial % 5)).astype(np.float32)
        if trial % 7 == 0:
            w = np.round(w * 64).astype(np.float32) / np.float32(64)   # coarse grid: many ties
        s16, z16, q = oracle.quantize_group(w, bits)
        assert list(q) == _brute_codes(w, s16, z16, bits)


@pytest.mark.parametrize("bits", [1, 2, 3])
def test_quantizer_scale_zero_properties(bits):
    """Levels span [min, max] up to the fp16 rounding of s and z; every value
    inside the span is within s/2 of its level; codes lie in [0, 2^b - 1]."""
    L = 2 ** bits - 1
    g = np.random.default_rng(20 + bits)
    for _ in range(200):
        w = (g.standard_normal(64) * g.uniform(0.001, 3.0) + g.uniform(-1, 1)).astype(np.float32)
        s16, z16, q = oracle.quantize_group(w, bits)
        s, z = f16val(s16), f16val(z16)
        mn, mx = float(w.min()), float(w.max())
        assert s > 0
        assert abs(s - (mx - mn) / L) <= 2.0 ** -10 * (mx - mn) / L + 1e-12
        assert q.max() <= L
        lo, hi = s * (0 - z), s * (L - z)
        tol = 2.0 ** -9 * (abs(mx) + abs(mn)) + 2.0 ** -11 * abs(z) * s * 4 + 1e-9
        assert abs(lo - mn) <= tol and abs(hi - mx) <= tol * (L + 1)
        for wi, qi in zip(w, q):
            if lo <= wi <= hi:
                assert abs(float(wi) - s * (int(qi) - z)) <= s / 2 * (1 + 1e-12)


def test_quantizer_golden_cases():
    for bits, vals, fill, s, z, codes in _lines("quant_ties.txt"):
        bits = int(bits)
        vals = [float(v) for v in vals.split()]
        w = np.full(32, float(fill), np.float32)
        w[: len(vals)] = vals
        s16, z16, q = oracle.quantize_group(w, bits)
        assert f16val(s16) == float(s)
        assert f16val(z16) == float(z) and not (z16 & 0x8000 and f16val(z16) == 0.0)
        assert list(q[: len(vals)]) == [int(c) for c in codes.split()]


def test_quantize_matrix_groups_along_rows():
    """Each row's groups are quantized independently (a transposed group axis fails)."""
    g = np.random.default_rng(3)
    W = (g.standard_normal((16, 128)) * 0.02).astype(np.float32)
    W[3, 64:96] *= 50.0                       # one loud group
    q, s, z = oracle.quantize(W, 2, 32)
    for r in range(16):
        for gi in range(4):
            s16, z16, qq = oracle.quantize_group(W[r, 32 * gi: 32 * gi + 32], 2)
            assert (s[r, gi], z[r, gi]) == (s16, z16)
            np.testing.assert_array_equal(q[r, 32 * gi: 32 * gi + 32], qq)
    assert f16val(s[3, 2]) > 20 * f16val(s[3, 1])


# ------------------------------------------------------------- dequant ---

def test_dequant_exact_and_single_rounding():
    """fp16 export = one RNE rounding of the exact rational s*(q - z) (numpy's
    float16 cast of the exact value); a naive fp32 product rounded again would
    differ on some of these triples."""
    g = np.random.default_rng(4)
    n = 200000
    s = (np.abs(g.standard_normal(n)) * 0.01 + 1e-4).astype(np.float16)
    z = (g.uniform(-1, 8, n)).astype(np.float16)
    q = g.integers(0, 8, n).astype(np.uint8)
    s16 = s.view(np.uint16).reshape(n, 1)
    z16 = z.view(np.uint16).reshape(n, 1)
    got = oracle.dequant_f16(q.reshape(n, 1), s16, z16, 1).ravel()
    exact = [Fraction(float(si)) * (int(qi) - Fraction(float(zi))) for si, zi, qi in zip(s, z, q)]
    want = np.array([float(v) for v in exact], np.float64).astype(np.float16).view(np.uint16)
    np.testing.assert_array_equal(got, want)


def test_dequant_double_rounding_cases():
    """Triples where an fp32 product rounded again to fp16 is one ulp off: the
    oracle must give the single rounding of the exact rational value."""
    for trip, good, bad in _lines("dequant_double_rounding.txt"):
        s16, z16, q = (int(v) for v in trip.split())
        exact = Fraction(f16val(s16)) * (q - Fraction(f16val(z16)))
        want = int(np.array([float(exact)]).astype(np.float16).view(np.uint16)[0])
        assert want == int(good) != int(bad)
        got = oracle.dequant_f16(np.array([[q]], np.uint8), np.array([[s16]], np.uint16),
                                 np.array([[z16]], np.uint16), 1)
        assert int(got[0, 0]) == want


# ---------------------------------------------------------------- layout ---

@pytest.mark.parametrize("bits", [1, 2, 3])
def test_layout_round_trip_and_size(bits):
    g = np.random.default_rng(5 + bits)
    R, K = 48, 384
    q = g.integers(0, 2 ** bits, (R, K)).astype(np.uint8)
    w = oracle.layout_pack(q, bits)
    assert w.size == R * K * bits // 32                 # dense: no padding words
    np.testing.assert_array_equal(oracle.layout_unpack(w, R, K, bits), q)
    # every bit of every word is used: all-ones codes give all-ones words
    full = oracle.layout_pack(np.full((R, K), 2 ** bits - 1, np.uint8), bits)
    assert (full == 0xFFFFFFFF).all()


def test_layout_golden_positions():
    for shape, code, words in _lines("layout_bits.txt"):
        R, K, bits = (int(v) for v in shape.split())
        n, k, c = (int(v) for v in code.split())
        q = np.zeros((R, K), np.uint8)
        q[n, k] = c
        w = oracle.layout_pack(q, bits)
        toks = words.split()
        want = {int(toks[i]): int(toks[i + 1], 16) for i in range(0, len(toks), 2)}
        nz = {int(i): int(w[i]) for i in np.nonzero(w)[0]}
        assert nz == want, (shape, code)


def test_scale_zero_layout():
    g = np.random.default_rng(6)
    R, K, G = 32, 256, 64
    s = g.integers(0, 65536, (R, K // G)).astype(np.uint16)
    z = g.integers(0, 65536, (R, K // G)).astype(np.uint16)
    sz = oracle.pack_sz(s, z, G)
    # closed form of the index: ((n/16)*(K/G) + g)*16 + n%16
    for n in (0, 5, 16, 31):
        for gi in range(K // G):
            idx = ((n // 16) * (K // G) + gi) * 16 + n % 16
            assert sz[idx] == int(s[n, gi]) | (int(z[n, gi]) << 16)
    s2, z2 = oracle.unpack_sz(sz, R, K, G)
    np.testing.assert_array_equal(s2, s)
    np.testing.assert_array_equal(z2, z)


# --------------------------------------------------------------- routing ---

def test_route_golden():
    rows = list(_lines("route_small.txt"))
    logits = np.array([[float(v) for v in r[0].split()] for r in rows], np.float32)
    imp = np.array([int(r[1]) for r in rows], np.uint8)
    out = oracle.route(logits, imp, 2, 0.3)
    for t, r in enumerate(rows):
        assert list(out["topk_idx"][t]) == [int(v) for v in r[2].split()]
        assert list(out["kept"][t]) == [int(v) for v in r[3].split()]
        np.testing.assert_allclose(out["topk_w"][t], [float(v) for v in r[4].split()], atol=1e-6)


def _naive_topk(l, k):
    return sorted(range(len(l)), key=lambda i: (-float(l[i]), i))[:k]


@pytest.mark.parametrize("cid,T", [(1, 64), (4, 300), (2, 32)])
def test_route_matches_naive_sort_and_softmax(cid, T):
    c = synthetic.config(cid)
    E, k, tau = c["E"], c["k"], c["tau"][0]
    lg = synthetic.logits(cid, T)
    lg[::7, 1] = lg[::7, 0]                  # exact ties
    imp = synthetic.important_mask(cid, T)
    out = oracle.route(lg, imp, k, tau)
    for t in range(T):
        sel = _naive_topk(lg[t], k)
        assert list(out["topk_idx"][t]) == sel
        p = scipy.special.softmax(lg[t, sel].astype(np.float64))
        for r in range(1, k):
            if imp[t]:
                assert out["kept"][t, r] == 1
            elif abs(p[r] - tau) > 1e-9:
                assert out["kept"][t, r] == (0 if p[r] < tau else 1), (t, r, p[r])
        assert out["kept"][t, 0] == 1
        keep = out["kept"][t].astype(bool)
        want_w = np.where(keep, p, 0.0) / p[keep].sum()
        np.testing.assert_allclose(out["topk_w"][t], want_w, rtol=1e-12, atol=1e-15)


def test_route_k2_gap_rule_equals_eq5_ratio():
    """Eq. 5 prunes the secondary expert when w1/w0 < mu; with mu = tau/(1-tau)
    that is the logit-gap rule, checked in exact rationals away from the boundary."""
    g = np.random.default_rng(7)
    T, E = 4000, 8
    lg = (g.standard_normal((T, E)) * 1.5).astype(np.float32)
    for tau in (0.1, 0.3, 0.45):
        out = oracle.route(lg, None, 2, tau)
        mu = tau / (1 - tau)
        for t in range(T):
            i0, i1 = out["topk_idx"][t]
            ratio = math.exp(float(lg[t, i1]) - float(lg[t, i0]))       # w1/w0
            if abs(ratio - mu) > 1e-6:
                assert out["kept"][t, 1] == (0 if ratio < mu else 1)


def test_route_tau_zero_and_all_protected_prune_nothing():
    lg = synthetic.logits(4, 256)
    for tau, imp in ((0.0, None), (0.9, np.ones(256, np.uint8))):
        out = oracle.route(lg, imp, 8, tau)
        assert out["n_pruned"] == 0 and out["kept"].all()


def test_route_csr_invariants():
    for cid, T in ((4, 2048), (1, 64), (2, 32)):
        c = synthetic.config(cid)
        lg = synthetic.logits(cid, T)
        out = oracle.route(lg, synthetic.important_mask(cid, T), c["k"], c["tau"][0])
        k, E = c["k"], c["E"]
        assert out["counts"].sum() == T * k - out["n_pruned"]
        assert out["offsets"][0] == 0 and (np.diff(out["offsets"]) == out["counts"]).all()
        seen = set()
        for e in range(E):
            toks = out["pair_token"][out["offsets"][e]: out["offsets"][e + 1]]
            assert (np.diff(toks) > 0).all()
            for p in range(out["offsets"][e], out["offsets"][e + 1]):
                t, r = out["pair_token"][p], out["pair_rank"][p]
                assert out["topk_idx"][t, r] == e and out["kept"][t, r]
                assert out["pair_pos"][t, r] == p and out["pair_w"][p] == out["topk_w"][t, r]
                seen.add((t, r))
        assert len(seen) == out["counts"].sum()
        assert ((out["pair_pos"] >= 0) == out["kept"].astype(bool)).all()


# --------------------------------------------------------------- forward ---

def _swiglu_numpy(X, logical_e, G):
    (qg, sg, zg), (qu, su, zu), (qd, sd, zd) = logical_e
    Wg = oracle.dequant_exact(qg, sg, zg, G)
    Wu = oracle.dequant_exact(qu, su, zu, G)
    Wd = oracle.dequant_exact(qd, sd, zd, G)
    a = X @ Wg.T
    return (a * scipy.special.expit(a) * (X @ Wu.T)) @ Wd.T


def _tiny_layer(E, bits, G=32, d=256, ffn=512, seed_cfg=1):
    mats = synthetic.layer_weights(seed_cfg, E=E, d=d, ffn=ffn)
    _, _, logical = oracle.pack_layer(mats, bits, G)
    return logical


def test_forward_single_expert_is_plain_swiglu():
    """E = 1, k = 1: Eq. 1 reduces to one SwiGLU FFN (numpy matmuls on the
    dequantized weights)."""
    logical = _tiny_layer(1, [2])
    x = synthetic.activations(1, 16)
    lg = np.zeros((16, 1), np.float32)
    rt = oracle.route(lg, None, 1, 0.3)
    y = oracle.moe_forward(x, rt, logical, 32)
    want = _swiglu_numpy(oracle.bf16_to_float64(x), logical[0], 32)
    np.testing.assert_allclose(y, want, rtol=1e-10, atol=1e-12)


def test_forward_dense_topk_when_nothing_pruned():
    """tau = 0 with every token protected = dense top-k MoE with softmax weights."""
    c = synthetic.config(1)
    logical = _tiny_layer(4, c["bits"])
    T = 24
    x = synthetic.activations(1, T)
    lg = synthetic.logits(1, T)
    rt = oracle.route(lg, np.ones(T, np.uint8), 2, 0.0)
    y = oracle.moe_forward(x, rt, logical, 32)
    X = oracle.bf16_to_float64(x)
    want = np.zeros_like(y)
    for t in range(T):
        sel = _naive_topk(lg[t], 2)
        p = scipy.special.softmax(lg[t, sel].astype(np.float64))
        for r, e in enumerate(sel):
            want[t] += p[r] * _swiglu_numpy(X[t: t + 1], logical[e], 32)[0]
    np.testing.assert_allclose(y, want, rtol=1e-10, atol=1e-12)


def test_forward_pruned_token_uses_primary_only():
    """A pruned k = 2 token's output is exactly its primary expert's output (Eq. 5)."""
    c = synthetic.config(1)
    logical = _tiny_layer(4, c["bits"])
    T = 64
    x = synthetic.activations(1, T)
    lg = synthetic.logits(1, T)
    rt = oracle.route(lg, None, 2, 0.3)
    y = oracle.moe_forward(x, rt, logical, 32)
    X = oracle.bf16_to_float64(x)
    pruned = np.nonzero(rt["kept"][:, 1] == 0)[0]
    assert len(pruned) > 3
    for t in pruned[:4]:
        e0 = rt["topk_idx"][t, 0]
        np.testing.assert_allclose(y[t], _swiglu_numpy(X[t: t + 1], logical[e0], 32)[0],
                                   rtol=1e-10, atol=1e-12)


def test_forward_rows_and_tokens_subset():
    c = synthetic.config(1)
    logical = _tiny_layer(4, c["bits"])
    x = synthetic.activations(1, 64)
    rt = oracle.route(synthetic.logits(1, 64), synthetic.important_mask(1, 64), 2, 0.3)
    full = oracle.moe_forward(x, rt, logical, 32)
    rows = [0, 7, 100, 255]
    toks = [3, 10, 63]
    part = oracle.moe_forward(x, rt, logical, 32, rows=rows, tokens=toks)
    np.testing.assert_array_equal(part, full[np.ix_(toks, rows)])


# ---------------------------------------------------------- residual stack ---

def _bf16_rne(v):
    """Round fp64 values to bfloat16 (nearest, ties to even) by exact fp64
    arithmetic on the two neighbouring bf16 values; returns bits.  Written
    here independently of the oracle's C rounding."""
    v = np.asarray(v, dtype=np.float64)
    m, e = np.frexp(np.abs(v))                     # |v| = m 2^e, m in [0.5, 1)
    q = np.ldexp(1.0, e - 8)                       # bf16 quantum at |v| (8 significant bits)
    k = np.floor(np.abs(v) / q)                    # exact: division by a power of two
    rem = np.abs(v) - k * q                        # exact
    up = (rem > q / 2) | ((rem == q / 2) & (k % 2 == 1))
    mag = (k + up) * q
    out = np.copysign(mag, v).astype(np.float32)   # exact: at most 9 significant bits
    return (out.view(np.uint32) >> 16).astype(np.uint16)


def test_bf16_rne_helper_matches_torch_where_fp32_is_exact():
    import torch
    g = np.random.default_rng(5)
    v = (g.standard_normal(20000) * 10.0 ** g.integers(-3, 4, 20000)).astype(np.float32).astype(np.float64)
    want = torch.from_numpy(v.astype(np.float32)).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(_bf16_rne(v), want)


def test_rms_norm_matches_torch_float64():
    """xn = bf16(h / sqrt(mean(h^2) + eps)) against torch's rms_norm in
    float64 (unit gain, eps = 1e-5), rounded by the exact helper above."""
    import torch
    x = synthetic.activations(1, 16, d=512)
    x[3] = synthetic.to_bf16_bits(np.full(512, 1e-3, np.float32))     # eps matters here
    got = oracle.rms_norm(x)
    h = torch.from_numpy(oracle.bf16_to_float64(x))
    ref = torch.nn.functional.rms_norm(h, (512,), eps=1e-5).numpy()
    np.testing.assert_array_equal(got, _bf16_rne(ref))
    ms = (oracle.bf16_to_float64(got) ** 2).mean(axis=1)
    assert np.all(np.abs(ms[np.arange(16) != 3] - 1.0) < 1e-2)


def test_stack_single_expert_is_numpy_residual_swiglu():
    """E = 1, k = 1 layers: h_{l+1} = bf16(h_l + SwiGLU_l(bf16(rms_norm(h_l)))),
    the norm by torch, the SwiGLU by numpy matmuls on dequantized weights and
    every rounding by the exact helper above."""
    import torch
    nl, T = 3, 12
    layers = []
    for l in range(nl):
        mats = synthetic.stack_layer_weights(5, l, E=1, d=256, ffn=512)
        _, _, logical = oracle.pack_layer(mats, [2 + l % 2], 32)
        rt = oracle.route(np.zeros((T, 1), np.float32), None, 1, 0.3)
        layers.append((rt, logical))
    x = synthetic.activations(1, T)
    got = oracle.moe_stack(x, layers, 32)
    h = oracle.bf16_to_float64(x)
    for l, (rt, logical) in enumerate(layers):
        xn = torch.nn.functional.rms_norm(torch.from_numpy(h), (256,), eps=1e-5).numpy()
        xn = oracle.bf16_to_float64(_bf16_rne(xn))
        want = _bf16_rne(h + _swiglu_numpy(xn, logical[0], 32))
        np.testing.assert_array_equal(got[l], want)
        h = oracle.bf16_to_float64(want)


def test_stack_zero_experts_are_identity():
    """All-zero weights quantize to zero codes with zero dequantized value, so
    each layer adds nothing and the residual stream passes through unchanged."""
    T, E = 10, 4
    zeros = [tuple(np.zeros((512, 256) if m < 2 else (256, 512), np.float32) for m in range(3))
             for _ in range(E)]
    _, _, logical = oracle.pack_layer(zeros, [1, 2, 3, 2], 32)
    layers = [(oracle.route(synthetic.stack_logits(5, l, T, E=E), None, 2, 0.3), logical)
              for l in range(2)]
    x = synthetic.activations(1, T)
    got = oracle.moe_stack(x, layers, 32)
    for h in got:
        np.testing.assert_array_equal(h, x)


def test_stack_tokens_are_independent():
    """Each token's path depends only on its own row and routing: a token
    subset gives the same rows as the full run."""
    T, E = 16, 4
    bits = [1, 2, 3, 2]
    layers = []
    for l in range(2):
        mats = synthetic.stack_layer_weights(5, l, E=E, d=256, ffn=512)
        _, _, logical = oracle.pack_layer(mats, bits, 32)
        rt = oracle.route(synthetic.stack_logits(5, l, T, E=E), synthetic.stack_mask(5, l, T), 2, 0.3)
        layers.append((rt, logical))
    x = synthetic.activations(1, T)
    full = oracle.moe_stack(x, layers, 32)
    toks = [0, 5, 15]
    part = oracle.moe_stack(x, layers, 32, tokens=toks)
    for a, b in zip(full, part):
        np.testing.assert_array_equal(a[toks], b)
    # the residual is really there: the output differs from the MoE output alone
    y0 = oracle.moe_forward(x, layers[0][0], layers[0][1], 32)
    assert not np.array_equal(full[0], oracle.bf16_round_array(y0))


# ------------------------------------------------------- Eq. 6 importance ---

def _causal_attention(g, H, L):
    """Random causal attention probabilities (row-softmax over keys j <= i), bf16 bits."""
    s = g.standard_normal((H, L, L))
    s[:, np.triu_indices(L, 1)[0], np.triu_indices(L, 1)[1]] = -np.inf
    p = np.exp(s - s.max(axis=2, keepdims=True))
    p /= p.sum(axis=2, keepdims=True)
    return oracle.bf16_round_array(p)


def test_importance_golden():
    rows = [l.split() for l in open(os.path.join(GOLD, "importance_small.txt")) if l[0] != "#" and l.strip()]
    A = np.array([[float(v) for v in r[1:]] for r in rows if r[0] == "attn"])[None]
    x = np.array([[float(v) for v in r[1:]] for r in rows if r[0] == "token"])
    want = [float(v) for r in rows if r[0] == "importance" for v in r[1:]]
    for r in rows:
        if r[0] == "rho":
            I, mask = oracle.token_importance(oracle.bf16_round_array(A), oracle.bf16_round_array(x), float(r[1]))
            np.testing.assert_allclose(I, want, rtol=1e-12)
            assert mask.tolist() == [int(v) for v in r[3:]]


def test_importance_closed_forms():
    """Self-attention only: column sums 1, I_j = ||t_j||_1 / (L - j).  All
    attention on the first token: I_0 = ||t_0||_1, every other I_j = 0."""
    g = np.random.default_rng(11)
    H, L, d = 3, 37, 16
    xb = oracle.bf16_round_array(g.standard_normal((L, d)))
    norms = np.abs(oracle.bf16_to_float64(xb)).sum(axis=1)
    one = oracle.bf16_round_array(np.ones(1))[0]
    A = np.zeros((H, L, L), np.uint16)
    A[:, np.arange(L), np.arange(L)] = one
    I, _ = oracle.token_importance(A, xb, 0.1)
    np.testing.assert_allclose(I, norms / (L - np.arange(L)), rtol=1e-14)
    A = np.zeros((H, L, L), np.uint16)
    A[:, :, 0] = one
    I, mask = oracle.token_importance(A, xb, 0.1)
    np.testing.assert_allclose(I[0], norms[0], rtol=1e-14)
    assert np.all(I[1:] == 0.0)
    # n = floor(0.1 * 37 + 1/2) = 4: token 0, then the zero-importance tokens 1, 2, 3 (lowest index)
    assert mask.tolist() == [1, 1, 1, 1] + [0] * (L - 4)


def test_importance_uniform_causal():
    """Uniform causal attention 1/(i+1) (rounded to bf16 here, so compared to
    the harmonic closed form at bf16 precision)."""
    L, d = 50, 8
    A = np.tril(np.ones((L, L))) / (np.arange(L)[:, None] + 1.0)
    g = np.random.default_rng(3)
    xb = oracle.bf16_round_array(g.standard_normal((L, d)))
    norms = np.abs(oracle.bf16_to_float64(xb)).sum(axis=1)
    I, _ = oracle.token_importance(oracle.bf16_round_array(A)[None], xb, 0.02)
    harm = np.array([sum(1.0 / (i + 1) for i in range(j, L)) for j in range(L)])
    np.testing.assert_allclose(I, norms * harm / (L - np.arange(L)), rtol=2 ** -8)


def test_importance_heads_and_triangle():
    """I over H heads = mean of the single-head I's (the head average); values
    above the diagonal are never read."""
    g = np.random.default_rng(5)
    H, L, d = 4, 29, 12
    A = _causal_attention(g, H, L)
    xb = oracle.bf16_round_array(g.standard_normal((L, d)))
    I, _ = oracle.token_importance(A, xb, 0.1)
    per = np.mean([oracle.token_importance(A[h:h + 1], xb, 0.1)[0] for h in range(H)], axis=0)
    np.testing.assert_allclose(I, per, rtol=1e-12)
    junk = A.copy()
    iu = np.triu_indices(L, 1)
    junk[:, iu[0], iu[1]] = 0x7f7f
    np.testing.assert_array_equal(oracle.token_importance(junk, xb, 0.1)[0], I)


@pytest.mark.parametrize("L,rho", [(1, 0.02), (50, 0.02), (100, 0.02), (333, 0.1), (64, 0.5)])
def test_importance_selection_brute_force(L, rho):
    g = np.random.default_rng(L)
    A = _causal_attention(g, 2, L)
    xb = oracle.bf16_round_array(g.standard_normal((L, 8)))
    I, mask = oracle.token_importance(A, xb, rho)
    n = int(np.floor(rho * L + 0.5))
    assert oracle.protect_count(L, rho) == n
    top = sorted(range(L), key=lambda j: (-I[j], j))[:n]
    assert np.flatnonzero(mask).tolist() == sorted(top)


def test_median_ratio_brute_force():
    import statistics
    g = np.random.default_rng(8)
    for T, E in ((1, 2), (7, 8), (64, 8), (100, 64)):
        lg = g.standard_normal((T, E)).astype(np.float32)
        lg[::3, 1] = lg[::3, 0]                      # ties keep a ratio of 1
        ratios = []
        for t in range(T):
            order = sorted(range(E), key=lambda e: (-float(lg[t, e]), e))
            ratios.append(math.exp(float(lg[t, order[1]]) - float(lg[t, order[0]])))
        assert oracle.median_ratio(lg) == pytest.approx(statistics.median(ratios), rel=1e-15)


# -------------------------------------------------------------------- PMQ ---

def _pmq_gold():
    sig, alloc = [], []
    for r in _lines("pmq_small.txt"):
        if r[0] == "significance":
            lg = np.array([[float(v) for v in row.split()] for row in r[1].split(";")], np.float32)
            sig.append((lg, int(r[2]), [float(v) for v in r[3].split()], [float(v) for v in r[4].split()]))
        else:
            eps = [[float(v) for v in row.split()] for row in r[3].split(";")]
            alloc.append(([float(v) for v in r[1].split()], [float(v) for v in r[2].split()], eps,
                          int(r[4]), [int(v) for v in r[5].split()], float(r[6]),
                          [float(v) for v in r[7].split()]))
    return sig, alloc


def test_pmq_significance_hand_example():
    """Sec. 3.2.1 frequencies and mean routing weights on a hand-worked case
    (including an exact tie between two logits, lower index first)."""
    sig, _ = _pmq_gold()
    for lg, k, phi, w in sig:
        got_phi, got_w = oracle.pmq_significance(lg, k)
        np.testing.assert_allclose(got_phi, phi, rtol=0, atol=0)
        np.testing.assert_allclose(got_w, w, rtol=1e-7, atol=1e-12)


def test_pmq_significance_sums():
    """Every token selects k experts whose weights sum to one."""
    for cid, T in ((2, 300), (4, 200)):
        c = synthetic.config(cid)
        phi, w = oracle.pmq_significance(synthetic.logits(cid, T), c["k"])
        assert phi.sum() == pytest.approx(c["k"], rel=1e-12)
        assert w.sum() == pytest.approx(1.0, rel=1e-12)
        assert (w <= phi + 1e-15).all() and (phi <= 1).all()


def test_pmq_allocate_hand_examples():
    _, alloc = _pmq_gold()
    for phi, w, eps, total, bits, obj, (a, b, gm) in alloc:
        for solve in (oracle.pmq_allocate_bruteforce, oracle.pmq_allocate):
            got = solve(phi, w, eps, total, alpha=a, beta=b, gamma=gm)
            assert got[0] == bits and got[1] == obj


def test_pmq_allocate_matches_enumeration():
    """The dynamic programme against the enumeration of every width vector,
    on random instances (including exactly tied objectives and infeasible
    totals)."""
    g = np.random.default_rng(11)
    for trial in range(150):
        E = int(g.integers(2, 8))
        phi = g.uniform(0, 1, E)
        w = g.uniform(0, 1, E) * phi
        eps = np.sort(g.uniform(0, 4, (E, 3)), axis=1)[:, ::-1]
        if trial % 5 == 0:
            eps[:] = eps[0]                      # identical experts: many exact ties
            phi[:] = phi[0]
            w[:] = w[0]
        total = int(g.integers(E, 3 * E + 1))
        a, b, gm = [(1, 1, 2), (1.5, 1.5, 2), (2, 1, 2), (1, 2, 2)][trial % 4]
        bf = oracle.pmq_allocate_bruteforce(phi, w, eps, total, a, b, gm)
        dp = oracle.pmq_allocate(phi, w, eps, total, a, b, gm)
        assert bf == dp, (trial, bf, dp)
        if bf is not None:
            assert sum(bf[0]) == total and 3 in bf[0] and 2 in bf[0]
        else:
            assert total < E + 3 or total > 3 * E - 1


def test_pmq_allocate_favours_significant_experts():
    """With equal errors, the more significant (frequent, heavily weighted)
    expert never gets fewer bits than a less significant one."""
    g = np.random.default_rng(3)
    for _ in range(30):
        E = 6
        phi = np.sort(g.uniform(0.05, 1, E))
        w = phi * 0.5
        eps = np.tile([4.0, 1.5, 0.5], (E, 1))
        bits, _ = oracle.pmq_allocate(phi, w, eps, 13)
        assert all(bits[i] <= bits[i + 1] for i in range(E - 1)), bits


# ------------------------------------------------------ sign binarization ---

def _sign_matrix(seed=4, R=32, K=256):
    g = np.random.default_rng(seed)
    W = (g.standard_normal((R, K)) * 0.02).astype(np.float32)
    W[0, :8] = 0.0
    W[1, :8] = -0.0
    W[2, :] = np.abs(W[2, :])
    return W


def test_sign_binarization_eq7_to_9():
    """B = sign(W) with sign(0) = +1 (Eq. 8); B~ = (B + 1)/2 (Eq. 9); the
    dequantized weight is the sign times the scale mean|W| (up to the fp16
    rounding of the stored 2 * mean|W|)."""
    W = _sign_matrix()
    q, s, z = oracle.quantize_sign(W, 32)
    B = np.where(W >= 0, 1, -1)                    # numpy: -0 >= 0 is True
    np.testing.assert_array_equal(2 * q.astype(int) - 1, B)
    assert (q[1, :8] == 1).all() and (q[0, :8] == 1).all()
    deq = oracle.dequant_exact(q, s, z, 32)
    mean_abs = float(np.abs(W.astype(np.float64)).mean())
    assert np.all(np.abs(np.abs(deq) - mean_abs) <= mean_abs * 2.0 ** -11)
    assert len(np.unique(np.abs(deq))) == 1
    np.testing.assert_array_equal(np.sign(deq), B)
    # the dequantized fp16 value is exactly half the stored scale
    np.testing.assert_array_equal(oracle.dequant_f16(q, s, z, 32).view(np.uint16) & 0x7fff,
                                  (s.max() - 0x400) * np.ones_like(q, dtype=np.uint16))


def test_sign_binarization_product_is_eq10():
    """x . (s B) = s * (sum of x where B~ = 1 - sum of x where B~ = 0), Eq. 10."""
    W = _sign_matrix(seed=9, R=16, K=128)
    q, s, z = oracle.quantize_sign(W, 32)
    deq = oracle.dequant_exact(q, s, z, 32)
    x = np.random.default_rng(2).standard_normal((5, 128))
    scale = abs(deq[0, 0])
    want = np.stack([scale * (x @ (q[i] == 1) - x @ (q[i] == 0)) for i in range(16)], axis=1)
    np.testing.assert_allclose(x @ deq.T, want, rtol=1e-12, atol=1e-14)


def test_pack_layer_mixed_methods():
    """A layer with a sign-binarized 1-bit expert beside RTN experts packs each
    expert by its own method; the RTN experts are unchanged."""
    mats = synthetic.layer_weights(1, E=3, d=256, ffn=512)
    words0, sz0, lg0 = oracle.pack_layer(mats, [1, 1, 2], 32)
    words1, sz1, lg1 = oracle.pack_layer(mats, [1, 1, 2], 32, methods=[1, 0, 0])
    for m in range(3):
        for a, b in zip(lg0[1][m], lg1[1][m]):
            np.testing.assert_array_equal(a, b)
        np.testing.assert_array_equal(lg1[0][m][2], 0x3800)
        np.testing.assert_array_equal(lg1[0][m][0], (mats[0][m] >= 0).astype(np.uint8))


# ----------------------------------------------------------- router GEMM ---

def _bf(v):
    """bf16 bit patterns of values that bfloat16 holds exactly."""
    a = np.asarray(v, dtype=np.float32)
    b = (a.view(np.uint32) >> 16).astype(np.uint16)
    assert ((b.astype(np.uint32) << 16).view(np.float32) == a).all()
    return b.reshape(1, -1)


def _nearest_f32(S: Fraction) -> int:
    """fp32 bits nearest to the rational S by exact distance, ties to an even
    significand, a zero sum as +0 (brute force over the neighbours)."""
    if S == 0:
        return 0
    f = np.float32(float(S))
    cands = {f, np.nextafter(f, np.float32(np.inf)), np.nextafter(f, np.float32(-np.inf))}
    best = None
    for c in cands:
        if not np.isfinite(c):
            continue
        dist = abs(Fraction(float(c)) - S)
        key = (dist, int(np.array(c, np.float32).view(np.uint32)) & 1)
        if best is None or key < best[0]:
            best = (key, c)
    return int(np.array(best[1], np.float32).view(np.uint32))


def _logit_bits(xv, wv):
    return int(oracle.router_logits(_bf(xv), _bf(wv)).view(np.uint32)[0, 0])


@pytest.mark.parametrize("x,w,want", [
    ([1, 1, 1], [2.0 ** 30, 1, -(2.0 ** 30)], 0x3F800000),        # cancellation: exactly 1
    ([1, 2 ** -12, 2 ** -40], [1, 2 ** -12, 2 ** -40], 0x3F800001),  # just above a midpoint
    ([1, 2 ** -12, 2 ** -40], [1, 2 ** -12, -(2 ** -40)], 0x3F800000),  # just below it
    ([1, 2 ** -12], [1, 2 ** -12], 0x3F800000),                    # exact tie, even is 1.0
    ([1, 2 ** -12, 2 ** -12], [1, 2 ** -11, 2 ** -12], 0x3F800002),   # 1 + 3 2^-24: tie, even is 1 + 2^-22
    ([-1, 2 ** -12, 2 ** -40], [1, -(2 ** -12), 2 ** -40], 0xBF800000),  # -(1 + 2^-24) + 2^-80 -> -1
    ([2 ** -75, 2 ** -125], [2 ** -75, 2 ** -125], 0x00000001),    # 2^-150 + 2^-250: subnormal rounds up
    ([2 ** -75], [2 ** -75], 0x00000000),                          # 2^-150 alone: tie to +0
    ([0.0, -0.0], [-3.0, 5.0], 0x00000000),                        # zero sum is +0
])
def test_router_logits_hand_cases(x, w, want):
    """Each logit is the exact sum rounded once to fp32: cancellation that a
    running fp32 sum loses, ties to even, and sums that fp64 rounds onto an
    fp32 midpoint (where a fp64-then-fp32 cast rounds the wrong way)."""
    assert _logit_bits(x, w) == want


def test_router_logits_nearest_by_exact_distance():
    """Random rows built to land near fp32 rounding boundaries, against the
    nearest fp32 of the rational sum found by brute force."""
    g = np.random.default_rng(5)
    for _ in range(300):
        n = int(g.integers(2, 24))
        e = g.integers(-30, 10, n)
        m = g.integers(128, 256, n) / 128.0
        xv = (m * 2.0 ** e * g.choice([-1, 1], n)).astype(np.float32)
        wv = (g.integers(128, 256, n) / 128.0 * 2.0 ** g.integers(-20, 5, n)).astype(np.float32)
        if g.random() < 0.5:
            xv *= np.float32(2.0 ** -45)       # the rest below fp64's resolution at 1
        xv[0], wv[0] = 1.0, 1.0
        if n > 2:
            xv[1], wv[1] = 2.0 ** -12, float(g.choice([-1, 1])) * 2.0 ** -12   # half an ulp of 1
        S = sum(Fraction(float(a)) * Fraction(float(b)) for a, b in zip(xv, wv))
        assert _logit_bits(xv, wv) == _nearest_f32(S)


def test_router_logits_matches_fp64_matmul():
    """Mixtral-shaped rows: within one fp32 ulp of numpy's fp64 product cast to
    fp32, and equal to it almost everywhere (a transposed operand fails)."""
    x = synthetic.activations(2, 6)
    w = synthetic.router_weights(2)
    got = oracle.router_logits(x, w)
    ref = (oracle.bf16_to_float64(x) @ oracle.bf16_to_float64(w).T).astype(np.float32)
    ulp = np.spacing(np.abs(ref))
    assert (np.abs(got - ref) <= ulp).all()
    assert (got == ref).mean() > 0.95
    assert 0.5 < float(got.std()) < 2.0                    # unit-variance logits by construction


# ------------------------------------------------------------------ GPTQ ---

def test_codes_for_matches_quantizer():
    """With the parameters the quantizer picked for the same values, the
    nearest-code helper gives the quantizer's own codes (tie-heavy groups)."""
    g = np.random.default_rng(11)
    for bits in (1, 2, 3):
        W = (g.standard_normal((64, 128)) * 0.02).astype(np.float32)
        W[:8] = np.round(W[:8] * 400) / 400                    # many values on level midpoints
        q, s, z = oracle.quantize(W, bits, 32)
        got = oracle.codes_for(W, np.repeat(s, 32, axis=1), np.repeat(z, 32, axis=1), bits)
        np.testing.assert_array_equal(got, q)


def _calib_h(N, K, tag=0):
    return oracle.gptq_hessian(synthetic.calibration(1, N, K, tag=tag))


def test_gptq_hessian_is_gram():
    """H = 2 X^T X: symmetric, and x^T H x = 2 ||X x||^2 for a random x."""
    X = synthetic.calibration(1, 300, 64)
    H = oracle.gptq_hessian(X)
    Xf = oracle.bf16_to_float64(X)
    v = np.random.default_rng(3).standard_normal(64)
    np.testing.assert_array_equal(H, H.T)
    assert np.isclose(v @ H @ v, 2 * np.sum((Xf @ v) ** 2), rtol=1e-12)


def test_gptq_factor_properties():
    """U is upper triangular with a positive diagonal and U^T U is the inverse
    of the damped H; scaling H by c scales U by 1/sqrt(c) (relative damping);
    a zero input row/column is dead and gets H_kk = 1 before damping."""
    H = _calib_h(200, 96)
    H[5, :] = 0.0
    H[:, 5] = 0.0
    U, dead = oracle.gptq_factor(H, 0.01)
    assert dead.tolist() == [1 if k == 5 else 0 for k in range(96)]
    np.testing.assert_array_equal(U, np.triu(U))
    assert (np.diag(U) > 0).all()
    Hd = H.copy()
    Hd[5, 5] = 1.0
    Hd[np.diag_indices(96)] += 0.01 * np.mean(np.diag(Hd))
    np.testing.assert_allclose(U.T @ U @ Hd, np.eye(96), atol=1e-9)
    U4, _ = oracle.gptq_factor(H * 4.0, 0.01)
    # dead H_kk is set to 1 regardless of scale, so compare without a dead input
    H2 = _calib_h(200, 96, tag=1)
    Ua, _ = oracle.gptq_factor(H2, 0.01)
    Ub, _ = oracle.gptq_factor(H2 * 4.0, 0.01)
    np.testing.assert_allclose(Ub, Ua / 2.0, rtol=1e-9, atol=1e-12)
    assert U4.shape == U.shape


def test_gptq_identity_hessian_is_rtn():
    """With H a multiple of I no error is passed on: GPTQ = the Sec. 3.1
    round-to-nearest quantizer bit for bit, loss = (h / 2) sum (w - deq)^2."""
    K, R = 128, 48
    c = 2.0 ** -3
    X = np.zeros((K, K), np.uint16)
    X[np.arange(K), np.arange(K)] = oracle.bf16_round(c)          # X = c I
    H = oracle.gptq_hessian(X)
    W = (np.random.default_rng(4).standard_normal((R, K)) * 0.02).astype(np.float32)
    for bits, G in ((1, 32), (2, 64), (3, 128)):
        q, s, z, loss, _ = oracle.gptq_quantize(W, H, bits, G)
        qr, sr, zr = oracle.quantize(W, bits, G)
        np.testing.assert_array_equal(q, qr)
        np.testing.assert_array_equal(s, sr)
        np.testing.assert_array_equal(z, zr)
        h = 2 * c * c * 1.01
        d = W.astype(np.float64) - oracle.dequant_exact(qr, sr, zr, G)
        np.testing.assert_allclose(loss, h / 2 * (d * d).sum(axis=1), rtol=1e-12)


def _nearest_exact(w32, s16, z16, bits):
    """Brute force over all codes with exact rationals, ties to the even code."""
    s, z = Fraction(f16val(s16)), Fraction(f16val(z16))
    best = None
    for j in range(1 << bits):
        key = (abs(Fraction(float(w32)) - s * (j - z)), j & 1)
        if best is None or key < best[0]:
            best = (key, j)
    return best[1]


def test_gptq_two_columns_closed_form():
    """K = 2, one group, H = [[1, rho], [rho, 1]], no damping: U = [[1/c, -rho/c],
    [0, 1]] with c = sqrt(1 - rho^2), so column 1 is quantized at
    w1 + rho (w0 - deq0) (optimal brain surgeon compensation), and the loss is
    ((w0 - deq0)^2 c^2 + (w1' - deq1)^2) / 2."""
    g = np.random.default_rng(8)
    for rho in (0.9, -0.6, 0.3):
        H = np.array([[1.0, rho], [rho, 1.0]])
        W = (g.standard_normal((40, 2)) * 0.05).astype(np.float32)
        for bits in (1, 2, 3):
            q, s, z, loss, _ = oracle.gptq_quantize(W, H, bits, 2, damp=0.0)
            for r in range(40):
                _, s16, z16 = oracle.quantize(W[r:r + 1], bits, 2)
                s16, z16 = int(s16[0, 0]), int(z16[0, 0])
                assert (s[r, 0], z[r, 0]) == (s16, z16)
                q0 = _nearest_exact(W[r, 0], s16, z16, bits)
                deq0 = f16val(s16) * (q0 - f16val(z16))
                w1 = float(W[r, 1]) + rho * (float(W[r, 0]) - deq0)
                q1 = _nearest_exact(np.float32(w1), s16, z16, bits)
                deq1 = f16val(s16) * (q1 - f16val(z16))
                assert (q[r, 0], q[r, 1]) == (q0, q1), (rho, bits, r)
                want = ((float(W[r, 0]) - deq0) ** 2 * (1 - rho * rho) + (w1 - deq1) ** 2) / 2
                assert math.isclose(loss[r], want, rel_tol=1e-12, abs_tol=1e-18)


def test_gptq_loss_identity():
    """Whatever codes are chosen, the error terms satisfy d H d^T = sum_k e_k^2
    per row (d = w - dequantized w, H the damped Hessian): a wrong sign, index
    or factor in the compensation breaks it."""
    K, R = 192, 32
    X = synthetic.calibration(1, 256, K, tag=2)
    H = oracle.gptq_hessian(X)
    W = synthetic.weight(1, 0, 1, shape=(R, K))
    for bits, G in ((1, 32), (3, 64)):
        q, s, z, loss, _ = oracle.gptq_quantize(W, H, bits, G)
        Hd = H + 0.01 * np.mean(np.diag(H)) * np.eye(K)
        d = W.astype(np.float64) - oracle.dequant_exact(q, s, z, G)
        np.testing.assert_allclose(np.einsum("rk,kj,rj->r", d, Hd, d), 2 * loss, rtol=1e-9)


def test_gptq_beats_rtn_on_correlated_inputs():
    """The layer-wise error ||(W - Q) X^T||^2 that GPTQ minimises greedily is
    well below round-to-nearest's on correlated calibration inputs."""
    K, R = 256, 64
    X = synthetic.calibration(1, 512, K, tag=3)
    Xf = oracle.bf16_to_float64(X)
    H = oracle.gptq_hessian(X)
    W = synthetic.weight(1, 1, 0, shape=(R, K))
    for bits, G in ((2, 32), (3, 128)):
        q, s, z, _, _ = oracle.gptq_quantize(W, H, bits, G)
        qr, sr, zr = oracle.quantize(W, bits, G)
        e_g = np.sum(((W - oracle.dequant_exact(q, s, z, G)) @ Xf.T) ** 2)
        e_r = np.sum(((W - oracle.dequant_exact(qr, sr, zr, G)) @ Xf.T) ** 2)
        assert e_g < 0.6 * e_r, (bits, e_g, e_r)


def test_gptq_dead_inputs():
    """Inputs the calibration never excites are zeroed: their weights do not
    change the result, and their codes are the nearest level to 0."""
    K, R, G = 128, 16, 32
    X = synthetic.calibration(1, 256, K, tag=4)
    X[:, [3, 70]] = 0
    H = oracle.gptq_hessian(X)
    W = synthetic.weight(1, 2, 0, shape=(R, K))
    W2 = W.copy()
    W2[:, [3, 70]] = 5.0
    a = oracle.gptq_quantize(W, H, 2, G)
    b = oracle.gptq_quantize(W2, H, 2, G)
    for u, v in zip(a[:4], b[:4]):
        np.testing.assert_array_equal(u, v)
    q, s, z = a[:3]
    for k in (3, 70):
        want = oracle.codes_for(np.zeros(R, np.float32), s[:, k // G], z[:, k // G], 2)
        np.testing.assert_array_equal(q[:, k], want)


def test_gptq_group_params_follow_compensation():
    """A factor whose only off-diagonal entry couples column 0 to column 2
    (U = I + a e_0 e_2^T): column 2 is quantized at w2 - a (w0 - deq0), and the
    second group's scale/zero come from that compensated value, not from w2."""
    g = np.random.default_rng(12)
    a = 0.75
    U = np.eye(4)
    U[0, 2] = a
    W = (g.standard_normal((30, 4)) * 0.05).astype(np.float32)
    q, s, z, loss, _ = oracle.gptq_quantize_u(W, U, np.zeros(4, np.uint8), 2, 2)
    differs = 0
    for r in range(30):
        _, s0, z0 = oracle.quantize(W[r:r + 1, :2], 2, 2)
        s0, z0 = int(s0[0, 0]), int(z0[0, 0])
        q0 = _nearest_exact(W[r, 0], s0, z0, 2)
        w2 = np.float32(float(W[r, 2]) - a * (float(W[r, 0]) - f16val(s0) * (q0 - f16val(z0))))
        _, s1, z1 = oracle.quantize(np.array([[w2, W[r, 3]]], np.float32), 2, 2)
        assert (s[r, 1], z[r, 1]) == (int(s1[0, 0]), int(z1[0, 0])), r
        assert q[r, 2] == _nearest_exact(w2, int(s1[0, 0]), int(z1[0, 0]), 2)
        _, s1o, _ = oracle.quantize(W[r:r + 1, 2:], 2, 2)
        differs += int(s1o[0, 0]) != s[r, 1]
    assert differs > 10          # the compensation does move the second group's range
