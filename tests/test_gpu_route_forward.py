"""GPU parity of mc_moe_route_forward (routing and Eq. 1 in one call)
against the two separate calls, mc_route_and_prune + mc_moe_forward, on the
same inputs: every routing buffer and y bit for bit (the routing buffers
start out filled with garbage, so an entry the one-call path fails to write
shows up), and the routing against the oracle.
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


def packed(mc, cid, E, d, ffn, bits, G):
    mats = synthetic.layer_weights(cid, E=E, d=d, ffn=ffn)
    L = mc.PackedLayer(E, d, ffn, bits, G)
    mc.pack(to_dev(np.stack([m[0] for m in mats])), to_dev(np.stack([m[1] for m in mats])),
            to_dev(np.stack([m[2] for m in mats])), L)
    torch.cuda.synchronize()
    return L


def garbage(r):
    for t in (r.topk_idx, r.topk_w, r.kept, r.counts, r.offsets, r.pair_token, r.pair_rank, r.pair_w, r.pair_pos,
              r.n_pruned):
        t.view(torch.uint8).fill_(0x5a)


ROUTING = ("topk_idx", "topk_w", "kept", "counts", "offsets", "pair_pos", "n_pruned")


def bits_of(t):
    a = t.cpu().numpy()
    return a.view(np.uint32) if a.dtype == np.float32 else a


@pytest.mark.parametrize("cid,E,k,d,ffn,G,T,tau,imp", [
    (1, 4, 2, 256, 512, 32, 1, 0.3, True),
    (1, 4, 2, 256, 512, 32, 5, 0.3, True),
    (1, 4, 2, 256, 512, 32, 16, 0.3, False),
    (1, 4, 2, 256, 512, 32, 17, 0.3, True),       # two 16-token blocks per workgroup
    (1, 4, 2, 256, 512, 32, 64, 0.0, True),       # largest fused batch, no pruning
    (1, 4, 2, 256, 512, 32, 65, 0.3, True),       # first batch routed by the routing kernels
    (1, 4, 2, 256, 512, 32, 130, 0.3, True),      # prefill path
    (4, 64, 8, 2048, 1024, 64, 16, 0.05, True),   # OLMoE-shaped: 64 experts, top-8
    (4, 64, 8, 2048, 1024, 64, 64, 0.05, False),
    (2, 8, 2, 512, 1024, 128, 32, 0.3, True),     # Mixtral's E, k, G at a smaller d, ffn
])
def test_route_forward_equals_two_calls(mc, cid, E, k, d, ffn, G, T, tau, imp):
    bits = [1 + (e * 7 + 3) % 3 for e in range(E)]
    bits[0], bits[1] = 3, 2
    L = packed(mc, cid, E, d, ffn, bits, G)
    x = to_dev(synthetic.activations(cid, T, d=d).view(np.int16))
    lg = synthetic.logits(cid, T, E=E)
    mask = synthetic.important_mask(cid, T) if imp else None
    lgd, md = to_dev(lg), (to_dev(mask) if imp else None)
    ws = torch.empty(mc.forward_workspace(T, E, k, d, ffn), dtype=torch.uint8, device="cuda")
    ra, rb = mc.Routing(T, E, k), mc.Routing(T, E, k)
    garbage(ra)
    garbage(rb)
    ya = torch.empty((T, d), dtype=torch.int16, device="cuda")
    yb = torch.empty((T, d), dtype=torch.int16, device="cuda")
    mc.route_and_prune(lgd, md, tau, ra)
    mc.moe_forward(x, ra, L, ya, ws)
    torch.cuda.synchronize()
    ws.fill_(0x33)
    mc.route_forward(x, lgd, md, tau, rb, L, yb, ws)
    torch.cuda.synchronize()
    for name in ROUTING:
        np.testing.assert_array_equal(bits_of(getattr(rb, name)), bits_of(getattr(ra, name)), err_msg=name)
    n = int(ra.offsets[-1].item())
    for name in ("pair_token", "pair_rank", "pair_w"):
        np.testing.assert_array_equal(bits_of(getattr(rb, name))[:n], bits_of(getattr(ra, name))[:n], err_msg=name)
    np.testing.assert_array_equal(yb.cpu().numpy(), ya.cpu().numpy())
    if k > 2:
        return          # k > 2 prunes in fp64 with different exp implementations (margins: routing tests)
    ref = oracle.route(lg, mask, k, tau)
    np.testing.assert_array_equal(rb.topk_idx.cpu().numpy(), ref["topk_idx"])
    np.testing.assert_array_equal(rb.kept.cpu().numpy(), ref["kept"])
    np.testing.assert_array_equal(rb.counts.cpu().numpy(), ref["counts"])
    np.testing.assert_array_equal(rb.pair_token.cpu().numpy()[:n], ref["pair_token"][:n])


def test_route_forward_rejects(mc):
    L = mc.PackedLayer(4, 256, 512, [1, 2, 3, 2], 32)
    r = mc.Routing(8, 4, 2)
    x = torch.zeros((8, 256), dtype=torch.int16, device="cuda")
    y = torch.empty_like(x)
    lg = torch.zeros((8, 4), dtype=torch.float32, device="cuda")
    ws = torch.empty(16, dtype=torch.uint8, device="cuda")
    with pytest.raises(mc.MCError):
        mc.route_forward(x, lg, None, 0.3, r, L, y, ws)                       # workspace too small
    ws = torch.empty(mc.forward_workspace(8, 4, 2, 256, 512), dtype=torch.uint8, device="cuda")
    with pytest.raises(mc.MCError):
        mc.route_forward(x, lg, None, 1.5, r, L, y, ws)                       # threshold outside [0, 1]
