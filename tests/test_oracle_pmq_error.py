"""Pins of the oracle's Sec. 3.2.2 reconstruction error (the errors Eq. 4
takes) and of its unquantized SwiGLU expert, against what the definition
fixes: a hand-computed token, the definition taken literally (the F-norm of
the difference of two whole-layer outputs, one with only expert e replaced by
its quantized weights), an expert no token keeps, and weights already on the
1-bit grid."""
import math

import numpy as np

import oracle
import synthetic


def test_dense_expert_hand_token():
    # g = x . (1, 0) = 1, u = x . (0, 1) = 2, h = silu(1) * 2, y = (2 h, -h)
    X = np.array([[1.0, 2.0]])
    Y = oracle.dense_expert_forward(X, [[1.0, 0.0]], [[0.0, 1.0]], [[2.0], [-1.0]])
    h = 2.0 / (1.0 + math.exp(-1.0))
    np.testing.assert_allclose(Y, [[2.0 * h, -h]], rtol=1e-15)
    # the down projection is linear in Wd
    g = np.random.default_rng(1)
    X = g.standard_normal((3, 8))
    Wg, Wu, Wd = g.standard_normal((5, 8)), g.standard_normal((5, 8)), g.standard_normal((8, 5))
    np.testing.assert_allclose(oracle.dense_expert_forward(X, Wg, Wu, 3.0 * Wd),
                               3.0 * oracle.dense_expert_forward(X, Wg, Wu, Wd), rtol=1e-13)


def _layer(E, d, ffn, T, k, seed):
    g = np.random.default_rng(seed)
    W = [(g.standard_normal((E, ffn, d)) * 0.02).astype(np.float32),
         (g.standard_normal((E, ffn, d)) * 0.02).astype(np.float32),
         (g.standard_normal((E, d, ffn)) * 0.02).astype(np.float32)]
    x = synthetic.activations(1, T, d=d)
    return W, x


def _layer_output(X, rt, W):
    """F = sum over kept ranks of w_r E_e(x_t), dense weights W[m][e]."""
    T, k = rt["topk_idx"].shape
    F = np.zeros((T, W[2].shape[1]))
    for t in range(T):
        for r in range(k):
            if rt["kept"][t, r]:
                e = rt["topk_idx"][t, r]
                F[t] += rt["topk_w"][t, r] * oracle.dense_expert_forward(X[t:t + 1], W[0][e], W[1][e], W[2][e])[0]
    return F


def test_pmq_error_is_the_definition():
    E, d, ffn, T, k, G = 3, 64, 64, 12, 2, 32
    W, x = _layer(E, d, ffn, T, k, 5)
    lg = synthetic.logits(1, T, E=E)
    rt = oracle.route(lg, None, k, 0.0)
    eps = oracle.pmq_expert_error(W[0], W[1], W[2], x, rt, G)
    X = oracle.bf16_to_float64(x)
    F = _layer_output(X, rt, W)
    for e in range(E):
        for b in (1, 2, 3):
            Wq = [m.copy().astype(np.float64) for m in W]
            for i in range(3):
                q, s, z = oracle.quantize(W[i][e], b, G)
                Wq[i][e] = oracle.dequant_exact(q, s, z, G)
            want = np.sqrt(((_layer_output(X, rt, Wq) - F) ** 2).sum())
            assert abs(eps[e, b - 1] - want) <= 1e-9 * want, (e, b, eps[e, b - 1], want)
    # coarser widths change the output more (not a theorem, but far from a tie here)
    assert np.all(eps[:, 0] > eps[:, 1]) and np.all(eps[:, 1] > eps[:, 2])


def test_pmq_error_unused_expert_is_zero():
    E, d, ffn, T, k, G = 4, 64, 64, 10, 2, 32
    W, x = _layer(E, d, ffn, T, k, 6)
    lg = synthetic.logits(1, T, E=E).copy()
    lg[:, 3] = -1e3                      # no token selects expert 3
    rt = oracle.route(lg, None, k, 0.0)
    assert rt["counts"][3] == 0
    eps = oracle.pmq_expert_error(W[0], W[1], W[2], x, rt, G)
    assert np.all(eps[3] == 0.0) and np.all(eps[:3] > 0.0)


def test_pmq_error_zero_on_the_one_bit_grid():
    # every group holds values from {0, 1/2}: the 1-bit quantizer reproduces
    # them exactly (s = 1/2, z = 0; a constant group gets s = 1 and an exact
    # level), so only the 2- and 3-bit errors are nonzero
    E, d, ffn, T, k, G = 2, 64, 64, 8, 2, 32
    g = np.random.default_rng(7)
    W = [(g.integers(0, 2, (E, ffn, d)) * 0.5).astype(np.float32),
         (g.integers(0, 2, (E, ffn, d)) * 0.5).astype(np.float32),
         (g.integers(0, 2, (E, d, ffn)) * 0.5).astype(np.float32)]
    x = synthetic.activations(1, T, d=d)
    rt = oracle.route(synthetic.logits(1, T, E=E), None, k, 0.0)
    eps = oracle.pmq_expert_error(W[0], W[1], W[2], x, rt, G)
    X = oracle.bf16_to_float64(x)
    scale = np.sqrt((_layer_output(X, rt, W) ** 2).sum())
    assert np.all(eps[:, 0] <= 1e-12 * scale), (eps, scale)
    assert np.all(eps[:, 1] > 1e-6 * scale)
