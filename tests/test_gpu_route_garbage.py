"""mc_moe_forward on routing buffers that no routing call filled (garbage):
every index the kernels take from them is range-checked on the device
(expert ranges, pair blocks, token and position clamps, the prefill set-up's
capacity check), so the call completes and writes y -- wrong values, but no
access outside a buffer.  Decode (32 tokens) and the grouped GEMMs (300
tokens, once with counts too large for the prefill tables and once with
counts that fit and garbage offsets).  tests/test_route_audit.py checks the
same index derivations on the CPU."""
import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def mc():
    import paper_2410_06270_amd as m
    m.load()
    return m


@pytest.mark.parametrize("T,fits", [(32, False), (300, False), (300, True)])
def test_forward_on_garbage_routing(mc, T, fits):
    E, d, ffn, k, G = 8, 512, 1024, 2, 128
    bits = [3, 2, 1, 2, 3, 3, 2, 1]
    gen = torch.Generator(device="cuda")
    gen.manual_seed(7 + T)
    w = [torch.randn((E, ffn, d) if m < 2 else (E, d, ffn), generator=gen, device="cuda").mul_(0.02)
         for m in range(3)]
    L = mc.PackedLayer(E, d, ffn, bits, G)
    mc.pack(w[0], w[1], w[2], L)
    r = mc.Routing(T, E, k)
    g = np.random.default_rng(T)
    P = T * k
    hi = 1 << 30

    def garbage(n):
        a = np.where(g.random(n) < 0.5, g.integers(-hi, hi, n), g.integers(-2 * P, 2 * P, n)).astype(np.int32)
        return torch.from_numpy(a).cuda()

    for buf in (r.counts, r.offsets, r.pair_token, r.pair_pos):
        buf.copy_(garbage(buf.numel()).view_as(buf))
    if fits:
        # counts the prefill tables can hold (the GEMMs run), offsets garbage
        r.counts.copy_(torch.from_numpy(g.integers(0, P // E + 1, E).astype(np.int32)).cuda())
    else:
        r.counts[:2] = P                    # two experts claim every pair slot
        r.offsets[:2] = 0
    r.topk_w.copy_(torch.from_numpy(g.random(r.topk_w.numel()).astype(np.float32)).view_as(r.topk_w).cuda())
    x = torch.randn((T, d), generator=gen, device="cuda").to(torch.bfloat16).view(torch.int16)
    y = torch.full((T, d), 0x7FC1, dtype=torch.int16, device="cuda")     # a NaN pattern no result has
    ws = torch.empty(mc.forward_workspace(T, E, k, d, ffn), dtype=torch.uint8, device="cuda")
    print("garbage routing T=%d fits=%d" % (T, fits), flush=True)
    mc.moe_forward(x, r, L, y, ws)
    torch.cuda.synchronize()
    assert not (y == 0x7FC1).any()          # every output written
