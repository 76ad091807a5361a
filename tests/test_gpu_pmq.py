"""The reconstruction error of Sec. 3.2.2 on the GPU (mc_pmq_expert_error)
against the oracle, and the whole PMQ chain of Sec. 3.2 through the C-ABI:
calibration logits -> significance (phi, w) -> errors -> the Eq. 4 widths ->
mc_pack -> the forward.  The GPU errors come from the packed forward's expert
kernels and dense fp32 kernels, the oracle's from fp64 arithmetic on the same
quantization: they agree to a relative 5e-3 (the forward's fp16 h is the
largest difference), and the widths chosen from them are identical.  Decode
(64 tokens) and grouped-GEMM (96 tokens) batches."""
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


@pytest.mark.parametrize("T", [64, 96])
def test_pmq_error_and_allocation(mc, T):
    c = synthetic.config(1)
    E, d, ffn, k, G = c["E"], c["d"], c["ffn"], c["k"], c["G"]
    mats = synthetic.layer_weights(1, E=E, d=d, ffn=ffn)
    W = [np.stack([m[i] for m in mats]) for i in range(3)]
    x = synthetic.activations(1, T)
    lg = synthetic.logits(1, T)
    rt = oracle.route(lg, None, k, 0.0)
    eps_ref = oracle.pmq_expert_error(W[0], W[1], W[2], x, rt, G)

    r = mc.Routing(T, E, k)
    mc.route_and_prune(to_dev(lg), None, 0.0, r)
    ws = torch.empty(mc.pmq_error_workspace(T, E, k, d, ffn, G), dtype=torch.uint8, device="cuda")
    wd = [to_dev(w) for w in W]
    print("pmq error T=%d" % T, flush=True)
    eps = mc.pmq_expert_error(wd[0], wd[1], wd[2], to_dev(x.view(np.int16)), r, G, ws)
    print("eps gpu", eps.tolist(), "\neps ref", eps_ref.tolist())
    np.testing.assert_allclose(eps, eps_ref, rtol=5e-3, atol=0)
    # a second call on the same workspace gives the same errors (nothing stale)
    eps2 = mc.pmq_expert_error(wd[0], wd[1], wd[2], to_dev(x.view(np.int16)), r, G, ws)
    np.testing.assert_array_equal(eps, eps2)

    # the chain: significance, the Eq. 4 widths at a 2-bit average, pack, forward
    phi, w = mc.pmq_significance(lg, k)
    phi_ref, w_ref = oracle.pmq_significance(lg, k)
    np.testing.assert_array_equal(phi, phi_ref)
    np.testing.assert_array_equal(w, w_ref)
    bits, _ = mc.pmq_allocate(phi, w, eps, 2 * E)
    bits_ref, _ = oracle.pmq_allocate(phi_ref, w_ref, eps_ref, 2 * E)
    assert list(bits) == list(bits_ref), (bits, bits_ref)
    assert sum(bits) == 2 * E and 3 in bits and 2 in bits
    L = mc.PackedLayer(E, d, ffn, bits, G)
    mc.pack(wd[0], wd[1], wd[2], L)
    y = torch.empty((T, d), dtype=torch.int16, device="cuda")
    fws = torch.empty(mc.forward_workspace(T, E, k, d, ffn), dtype=torch.uint8, device="cuda")
    mc.moe_forward(to_dev(x.view(np.int16)), r, L, y, fws)
    torch.cuda.synchronize()
    _, _, logical = oracle.pack_layer(mats, bits, G)
    y_ref = oracle.moe_forward(x, rt, logical, G)
    g = oracle.bf16_to_float64(y.cpu().numpy().view(np.uint16))
    rb = oracle.bf16_to_float64(oracle.bf16_round_array(y_ref))
    assert np.abs(g - rb).mean() <= 1e-3
