"""GPU parity of the GPTQ quantizer (Hessian, factor, in-order quantization
into the packed layer) through the C-ABI against the oracle.

* Hessian: H = 2 X^T X in fp64 from the same bf16 inputs; products are exact,
  so the two sums differ only by fp64 summation order: |dH| <= N 2^-52
  sum_t |x_ti x_tj| elementwise.  The GPU result is exactly symmetric.
* Factor: U from the oracle's H, within 1e-10 max|U| (fp64 factorizations of
  a damped Gram matrix; condition numbers here are below 1e4).
* Quantize: given the oracle's U and dead mask, the kernel applies the same
  fp64 operations in the same order (per-column updates, each product and
  subtraction rounded), so codes, scale/zero words and packed words are equal
  bit for bit and the per-row loss is equal up to its summation order.
* End to end (the GPU's own H and U): codes equal on almost every row; the
  layer-wise error ||(W - Q) X^T||^2 within 1e-6 of the oracle's.
"""
import numpy as np
import pytest

import oracle
import synthetic

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def mc():
    import paper_2410_06270_amd as m
    m.load()
    return m


def to_dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def gpu_hessian(mc, X, accumulate_from=None):
    K = X.shape[1]
    H = torch.zeros((K, K), dtype=torch.float64, device="cuda") if accumulate_from is None else accumulate_from
    mc.gptq_hessian(to_dev(X.view(np.int16)), H, accumulate=accumulate_from is not None)
    torch.cuda.synchronize()
    return H


def gpu_factor(mc, H, damp=0.01, R=16):
    K = H.shape[0]
    U = torch.empty((K, K), dtype=torch.float64, device="cuda")
    dead = torch.empty(K, dtype=torch.uint8, device="cuda")
    ws = torch.empty(mc.gptq_workspace(R, K), dtype=torch.uint8, device="cuda")
    mc.gptq_factor(H, U, dead, ws, damp=damp)
    torch.cuda.synchronize()
    return U, dead


def rtn_layer(mc, mats, bits, G):
    E = len(mats)
    ffn, d = mats[0][0].shape
    L = mc.PackedLayer(E, d, ffn, bits, G)
    mc.pack(to_dev(np.stack([m[0] for m in mats])), to_dev(np.stack([m[1] for m in mats])),
            to_dev(np.stack([m[2] for m in mats])), L)
    torch.cuda.synchronize()
    return L


def gpu_quantize(mc, L, e, m, W, U, dead):
    R, K = W.shape
    ws = torch.empty(mc.gptq_workspace(R, K), dtype=torch.uint8, device="cuda")
    loss = torch.empty(R, dtype=torch.float64, device="cuda")
    mc.gptq_quantize(L, e, m, to_dev(W), U, dead, ws, loss=loss)
    torch.cuda.synchronize()
    return loss.cpu().numpy()


def export_codes(mc, L, e, m, R, K):
    out = torch.empty((R, K), dtype=torch.uint8, device="cuda")
    mc.codes_export(L, e, m, out)
    torch.cuda.synchronize()
    return out.cpu().numpy()


def matrix_words(L, bits, G, e, m):
    """(words, sz) slices of matrix m of expert e, from the layer offsets."""
    E, d, ffn = L.E, L.d, L.ffn
    wofs, sofs, _, _ = oracle.layer_offsets(E, d, ffn, bits, G)
    R, K = (ffn, d) if m < 2 else (d, ffn)
    words = L.words.cpu().numpy().view(np.uint32)
    sz = L.sz.cpu().numpy().view(np.uint32)
    nw = R * K * bits[e] // 32
    ns = R * K // G
    return words[wofs[(e, m)]:wofs[(e, m)] + nw], sz[sofs[(e, m)]:sofs[(e, m)] + ns]


@pytest.mark.parametrize("N,K", [(300, 256), (1000, 640)])
def test_gptq_hessian(mc, N, K):
    X = synthetic.calibration(1, N, K, tag=N)
    H = gpu_hessian(mc, X).cpu().numpy()
    ref = oracle.gptq_hessian(X)
    Xa = np.abs(oracle.bf16_to_float64(X))
    bound = N * 2.0 ** -52 * 2.0 * (Xa.T @ Xa)
    assert (np.abs(H - ref) <= bound).all()
    np.testing.assert_array_equal(H, H.T)
    # calibration in two pieces
    Hp = gpu_hessian(mc, X[: N // 3])
    Hp = gpu_hessian(mc, X[N // 3:], accumulate_from=Hp).cpu().numpy()
    assert (np.abs(Hp - ref) <= 2 * bound).all()


@pytest.mark.parametrize("K,dead_cols", [(256, []), (512, [7, 300])])
def test_gptq_factor(mc, K, dead_cols):
    X = synthetic.calibration(1, 2 * K, K, tag=K)
    X[:, dead_cols] = 0
    H = oracle.gptq_hessian(X)
    U, dead = gpu_factor(mc, to_dev(H))
    Ur, deadr = oracle.gptq_factor(H)
    np.testing.assert_array_equal(dead.cpu().numpy(), deadr)
    U = U.cpu().numpy()
    np.testing.assert_array_equal(U, np.triu(U))
    assert np.abs(U - Ur).max() <= 1e-10 * np.abs(Ur).max()


CASES = [  # (E, d, ffn, bits, G, expert, matrix)
    (2, 256, 512, [2, 3], 32, 0, 0),
    (2, 256, 512, [1, 3], 64, 0, 1),
    (2, 256, 512, [2, 3], 128, 1, 2),
    (3, 384, 640, [3, 1, 2], 128, 1, 2),      # K = 640: five column blocks, d = 384
    (2, 256, 512, [1, 2], 32, 0, 2),
]


@pytest.mark.parametrize("E,d,ffn,bits,G,e,m", CASES)
def test_gptq_quantize_bit_exact(mc, E, d, ffn, bits, G, e, m):
    mats = synthetic.layer_weights(1, E=E, d=d, ffn=ffn)
    W = mats[e][m]
    R, K = W.shape
    X = synthetic.calibration(1, 2 * K, K, tag=K + m)
    X[:, 5] = 0                                   # one dead input
    U, dead = oracle.gptq_factor(oracle.gptq_hessian(X))
    q, s, z, loss, margin = oracle.gptq_quantize_u(W, U, dead, bits[e], G)
    L = rtn_layer(mc, mats, bits, G)
    got_loss = gpu_quantize(mc, L, e, m, W, to_dev(U), to_dev(dead))
    codes = export_codes(mc, L, e, m, R, K)
    words, sz = matrix_words(L, bits, G, e, m)
    same = (codes == q).all(axis=1)
    assert (same | (margin < 1e-12)).all(), np.flatnonzero(~same)[:8]
    rows = np.flatnonzero(same)
    assert len(rows) >= R - 2
    if same.all():
        np.testing.assert_array_equal(words, oracle.layout_pack(q, bits[e]))
        np.testing.assert_array_equal(sz, oracle.pack_sz(s, z, G))
    np.testing.assert_allclose(got_loss[rows], loss[rows], rtol=1e-12)
    # the other matrices keep their round-to-nearest packing
    _, _, logical = oracle.pack_layer(mats, bits, G)
    for ee in range(E):
        for mm in range(3):
            if (ee, mm) == (e, m):
                continue
            qq, ss, zz = logical[ee][mm]
            ww, sw = matrix_words(L, bits, G, ee, mm)
            np.testing.assert_array_equal(ww, oracle.layout_pack(qq, bits[ee]))
            np.testing.assert_array_equal(sw, oracle.pack_sz(ss, zz, G))


def test_gptq_end_to_end(mc):
    """The GPU's own Hessian and factor: codes equal on almost every row, the
    layer-wise error equal to the oracle's, and well below round-to-nearest."""
    E, d, ffn, bits, G = 2, 512, 1024, [2, 3], 128
    mats = synthetic.layer_weights(1, E=E, d=d, ffn=ffn)
    W = mats[0][0]
    R, K = W.shape
    X = synthetic.calibration(1, 2048, K, tag=99)
    H = gpu_hessian(mc, X)
    U, dead = gpu_factor(mc, H)
    L = rtn_layer(mc, mats, bits, G)
    gpu_quantize(mc, L, 0, 0, W, U, dead)
    codes = export_codes(mc, L, 0, 0, R, K)
    q, s, z, _, _ = oracle.gptq_quantize(W, oracle.gptq_hessian(X), bits[0], G)
    assert (codes == q).all(axis=1).mean() >= 0.95
    Xf = oracle.bf16_to_float64(X)
    deq = torch.empty((R, K), dtype=torch.int16, device="cuda")
    mc.dequant_export(L, 0, 0, deq)
    torch.cuda.synchronize()
    wq = deq.cpu().numpy().view(np.uint16).view(np.float16).astype(np.float64)
    err_gpu = np.sum(((W - wq) @ Xf.T) ** 2)
    err_ref = np.sum(((W - oracle.dequant_f16(q, s, z, G).view(np.float16).astype(np.float64)) @ Xf.T) ** 2)
    assert abs(err_gpu - err_ref) <= 1e-6 * err_ref
    qr, sr, zr = oracle.quantize(W, bits[0], G)
    err_rtn = np.sum(((W - oracle.dequant_exact(qr, sr, zr, G)) @ Xf.T) ** 2)
    assert err_gpu < 0.6 * err_rtn


def test_gptq_rejects(mc):
    L = mc.PackedLayer(2, 256, 512, [2, 3], 32)
    ws = torch.empty(16, dtype=torch.uint8, device="cuda")
    W = torch.zeros((512, 256), dtype=torch.float32, device="cuda")
    U = torch.zeros((256, 256), dtype=torch.float64, device="cuda")
    dead = torch.zeros(256, dtype=torch.uint8, device="cuda")
    with pytest.raises(mc.MCError):
        mc.gptq_quantize(L, 0, 0, W, U, dead, ws)          # workspace too small
    with pytest.raises(mc.MCError):
        mc.gptq_quantize(L, 2, 0, W, U, dead, ws)          # no expert 2


def _sample_rows(R, n=12, seed=0):
    g = np.random.default_rng(seed)
    return sorted({0, R - 1, *g.choice(R, n - 2, replace=False).tolist()})


def test_gptq_fullsize_mixtral_gate(mc):
    """Mixtral expert gate matrix (14336 x 4096, 3 bits, G = 128) from 8192
    calibration rows, entirely on the GPU; sampled rows against the oracle's
    own pipeline (its H, its U)."""
    d, ffn, G, bits = 4096, 14336, 128, 3
    W = synthetic.weight(2, 0, 0, shape=(ffn, d))
    X = synthetic.calibration(2, 8192, d, tag=1)
    H = gpu_hessian(mc, X)
    U, dead = gpu_factor(mc, H, R=ffn)
    L = mc.PackedLayer(1, d, ffn, [bits], G)
    mc.pack(to_dev(W[None]), to_dev(W[None]), to_dev(synthetic.weight(2, 0, 2, shape=(d, ffn))[None]), L)
    loss = gpu_quantize(mc, L, 0, 0, W, U, dead)
    codes = export_codes(mc, L, 0, 0, ffn, d)
    rows = _sample_rows(ffn)
    Ur, deadr = oracle.gptq_factor(oracle.gptq_hessian(X))
    q, s, z, lr, _ = oracle.gptq_quantize_u(W[rows], Ur, deadr, bits, G)
    same = (codes[rows] == q).all(axis=1)
    assert same.mean() >= 0.9, same
    np.testing.assert_allclose(loss[rows][same], lr[same], rtol=1e-9)


def test_gptq_fullsize_mixtral_down_loss_identity(mc):
    """Mixtral expert down matrix (4096 x 14336, 2 bits): on sampled rows the
    GPU's codes satisfy d H_d d^T = 2 loss with H_d = 2 X^T X + damping (the
    identity ties the factor, the codes and the compensation together), and
    the layer-wise error is below round-to-nearest's."""
    d, ffn, G, bits = 4096, 14336, 128, 2
    W = synthetic.weight(2, 0, 2, shape=(d, ffn))
    X = synthetic.calibration(2, 2048, ffn, tag=2)
    H = gpu_hessian(mc, X)
    U, dead = gpu_factor(mc, H, R=d)
    assert int(dead.sum().item()) == 0
    L = mc.PackedLayer(1, d, ffn, [bits], G)
    wg = synthetic.weight(2, 0, 0, shape=(ffn, d))
    mc.pack(to_dev(wg[None]), to_dev(wg[None]), to_dev(W[None]), L)
    loss = gpu_quantize(mc, L, 0, 2, W, U, dead)
    rows = _sample_rows(d)
    deq = torch.empty((d, ffn), dtype=torch.int16, device="cuda")
    mc.dequant_export(L, 0, 2, deq)
    torch.cuda.synchronize()
    codes = export_codes(mc, L, 0, 2, d, ffn)
    words, sz = matrix_words(L, [bits], G, 0, 2)
    s, z = oracle.unpack_sz(sz, d, ffn, G)
    Xf = oracle.bf16_to_float64(X)
    delta = W[rows].astype(np.float64) - oracle.dequant_exact(codes[rows], s[rows], z[rows], G)
    damp_add = 0.01 * np.mean(2.0 * np.sum(Xf * Xf, axis=0))
    quad = 2.0 * np.sum((Xf @ delta.T) ** 2, axis=0) + damp_add * np.sum(delta * delta, axis=1)
    np.testing.assert_allclose(quad, 2.0 * loss[rows], rtol=1e-6)
    qr, sr, zr = oracle.quantize(W[rows], bits, G)
    rtn = W[rows].astype(np.float64) - oracle.dequant_exact(qr, sr, zr, G)
    assert np.sum((Xf @ delta.T) ** 2) < 0.7 * np.sum((Xf @ rtn.T) ** 2)
