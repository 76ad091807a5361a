"""GPU parity of the residual MoE stack (mc_moe_stack_forward) against the oracle.

Each layer is checked on its own: the GPU runs layer l on the oracle's bf16
input h_l and its output is compared with the oracle's h_{l+1} =
bf16(h_l + Eq. 1 of layer l on RMSNorm(h_l)), so rounding differences do not
compound over layers.  Tolerance as for one layer (bf16 outputs, fp64 oracle): MAE of
|y - bf16(ref)| <= 1e-3 and max |y - ref| / max(|ref|, rms(ref)) <= 2e-2.
The n-layer call itself is checked to equal the chain of one-layer calls bit
for bit, at small shapes and at the Mixtral shape."""
import numpy as np
import pytest

import oracle
import synthetic

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")

TAU = 0.3


@pytest.fixture(scope="module")
def mc():
    import paper_2410_06270_amd as m
    m.load()
    return m


def to_dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def pack_layer_gpu(mc, E, d, ffn, bits, G, expert_mats):
    """Pack a layer from fp32 weights produced one expert at a time."""
    wg = torch.empty((E, ffn, d), dtype=torch.float32, device="cuda")
    wu = torch.empty((E, ffn, d), dtype=torch.float32, device="cuda")
    wd = torch.empty((E, d, ffn), dtype=torch.float32, device="cuda")
    for e in range(E):
        g, u, dn = expert_mats(e)
        wg[e].copy_(torch.from_numpy(g))
        wu[e].copy_(torch.from_numpy(u))
        wd[e].copy_(torch.from_numpy(dn))
    L = mc.PackedLayer(E, d, ffn, bits, G)
    mc.pack(wg, wu, wd, L)
    torch.cuda.synchronize()
    del wg, wu, wd
    torch.cuda.empty_cache()
    return L


def run_stack(mc, x_bits, layers, logits, masks, k, E, d, ffn):
    """One mc_moe_stack_forward call; returns the bf16 bits of y."""
    T = x_bits.shape[0]
    r = mc.Routing(T, E, k)
    y = torch.empty((T, d), dtype=torch.int16, device="cuda")
    tmp = torch.empty((T, d), dtype=torch.int16, device="cuda") if len(layers) > 1 else None
    ws = torch.empty(mc.stack_workspace(T, E, k, d, ffn), dtype=torch.uint8, device="cuda")
    mc.stack_forward(to_dev(x_bits.view(np.int16)), layers, to_dev(np.stack(logits)),
                     to_dev(np.stack(masks)), TAU, r, y, tmp, ws)
    torch.cuda.synchronize()
    return y.cpu().numpy().view(np.uint16)


def check_layer(g_bits, h_in_bits, Y):
    """g_bits: GPU output rows; h_in_bits: the oracle's input rows; Y: the
    oracle's fp64 MoE output of those rows."""
    ref = oracle.bf16_to_float64(h_in_bits) + Y
    g = oracle.bf16_to_float64(g_bits)
    rb = oracle.bf16_to_float64(oracle.bf16_round_array(ref))
    mae = float(np.abs(g - rb).mean())
    rms = float(np.sqrt((ref ** 2).mean()))
    maxrel = float((np.abs(g - ref) / np.maximum(np.abs(ref), rms)).max())
    return mae, maxrel


SMALL = dict(E=8, d=512, ffn=1024, G=128, k=2)


@pytest.fixture(scope="module")
def small_stack(mc):
    E, d, ffn, G = SMALL["E"], SMALL["d"], SMALL["ffn"], SMALL["G"]
    out = []
    for l in range(4):
        bits = synthetic.stack_bits(5, l)
        mats = synthetic.stack_layer_weights(5, l, E=E, d=d, ffn=ffn)
        _, _, logical = oracle.pack_layer(mats, bits, G)
        L = pack_layer_gpu(mc, E, d, ffn, bits, G, lambda e: mats[e])
        out.append((bits, logical, L))
    return out


@pytest.mark.parametrize("T", [1, 8, 64, 130])
def test_stack_small_per_layer(mc, small_stack, T):
    E, d, ffn, G, k = SMALL["E"], SMALL["d"], SMALL["ffn"], SMALL["G"], SMALL["k"]
    x = synthetic.activations(1, T, d=d)
    h = x
    for l, (bits, logical, L) in enumerate(small_stack):
        lg = synthetic.stack_logits(5, l, T, E=E)
        mask = synthetic.stack_mask(5, l, T)
        rt = oracle.route(lg, mask, k, TAU)
        Y = oracle.moe_forward(oracle.rms_norm(h), rt, logical, G)
        g = run_stack(mc, h, [L], [lg], [mask], k, E, d, ffn)
        mae, maxrel = check_layer(g, h, Y)
        print("T=%d layer %d MAE %.3e MaxRel %.3e" % (T, l, mae, maxrel))
        assert mae <= 1e-3 and maxrel <= 2e-2, (l, mae, maxrel)
        h = oracle.moe_stack(h, [(rt, logical)], G)[0]


@pytest.mark.parametrize("T", [8, 130])
def test_stack_call_equals_chain_of_layers(mc, small_stack, T):
    E, d, ffn, k = SMALL["E"], SMALL["d"], SMALL["ffn"], SMALL["k"]
    x = synthetic.activations(1, T, d=d)
    lgs = [synthetic.stack_logits(5, l, T, E=E) for l in range(4)]
    masks = [synthetic.stack_mask(5, l, T) for l in range(4)]
    Ls = [s[2] for s in small_stack]
    whole = run_stack(mc, x, Ls, lgs, masks, k, E, d, ffn)
    h = x
    for l in range(4):
        h = run_stack(mc, h, [Ls[l]], [lgs[l]], [masks[l]], k, E, d, ffn)
    np.testing.assert_array_equal(whole, h)
    three = run_stack(mc, x, Ls[:3], lgs[:3], masks[:3], k, E, d, ffn)   # odd layer count
    h3 = x
    for l in range(3):
        h3 = run_stack(mc, h3, [Ls[l]], [lgs[l]], [masks[l]], k, E, d, ffn)
    np.testing.assert_array_equal(three, h3)


@pytest.mark.parametrize("T,n", [(1, 8), (8, 11), (64, 17), (130, 9)])
def test_stack_many_layers_equals_chain(mc, small_stack, T, n):
    """More layers than one routing launch covers (small batches route 8
    layers at a time, each into its own buffers, the last layer into r): the
    n-layer call equals the chain of one-layer calls bit for bit, and r then
    holds the last layer's routing as mc_route_and_prune writes it.  The four
    packed layers are reused in turn; every layer has its own logits and
    protected tokens."""
    E, d, ffn, k = SMALL["E"], SMALL["d"], SMALL["ffn"], SMALL["k"]
    x = synthetic.activations(1, T, d=d)
    lgs = [synthetic.stack_logits(5, l, T, E=E) for l in range(n)]
    masks = [synthetic.stack_mask(5, l, T) for l in range(n)]
    Ls = [small_stack[l % 4][2] for l in range(n)]
    r = mc.Routing(T, E, k)
    y = torch.empty((T, d), dtype=torch.int16, device="cuda")
    tmp = torch.empty((T, d), dtype=torch.int16, device="cuda")
    ws = torch.empty(mc.stack_workspace(T, E, k, d, ffn), dtype=torch.uint8, device="cuda")
    mc.stack_forward(to_dev(x.view(np.int16)), Ls, to_dev(np.stack(lgs)), to_dev(np.stack(masks)), TAU, r, y,
                     tmp, ws)
    torch.cuda.synchronize()
    whole = y.cpu().numpy().view(np.uint16)
    h = x
    for l in range(n):
        h = run_stack(mc, h, [Ls[l]], [lgs[l]], [masks[l]], k, E, d, ffn)
    np.testing.assert_array_equal(whole, h)
    ref = mc.Routing(T, E, k)
    mc.route_and_prune(to_dev(lgs[-1]), to_dev(masks[-1]), TAU, ref)
    torch.cuda.synchronize()
    P = int(ref.offsets[E].item())
    for name in ("topk_idx", "topk_w", "kept", "counts", "offsets", "pair_pos", "n_pruned"):
        assert torch.equal(getattr(r, name), getattr(ref, name)), name
    for name in ("pair_token", "pair_rank", "pair_w"):
        assert torch.equal(getattr(r, name)[:P], getattr(ref, name)[:P]), name


@pytest.mark.parametrize("T", [8, 130])
def test_stack_without_flags_equals_zero_flags(mc, small_stack, T):
    """important = NULL means no protected token: 10 layers (two routing
    launches for small batches) give the same bits as all-zero flags."""
    E, d, ffn, k = SMALL["E"], SMALL["d"], SMALL["ffn"], SMALL["k"]
    n = 10
    x = to_dev(synthetic.activations(1, T, d=d).view(np.int16))
    lgs = to_dev(np.stack([synthetic.stack_logits(5, l, T, E=E) for l in range(n)]))
    Ls = [small_stack[l % 4][2] for l in range(n)]
    outs = []
    for flags in (None, to_dev(np.zeros((n, T), np.uint8))):
        r = mc.Routing(T, E, k)
        y = torch.empty((T, d), dtype=torch.int16, device="cuda")
        tmp = torch.empty((T, d), dtype=torch.int16, device="cuda")
        ws = torch.empty(mc.stack_workspace(T, E, k, d, ffn), dtype=torch.uint8, device="cuda")
        mc.stack_forward(x, Ls, lgs, flags, TAU, r, y, tmp, ws)
        torch.cuda.synchronize()
        outs.append(y.cpu().numpy())
    np.testing.assert_array_equal(outs[0], outs[1])


def test_stack_rejects_aliased_buffers(mc, small_stack):
    E, d, ffn, k = SMALL["E"], SMALL["d"], SMALL["ffn"], SMALL["k"]
    T = 4
    r = mc.Routing(T, E, k)
    x = torch.zeros((T, d), dtype=torch.int16, device="cuda")
    ws = torch.empty(mc.stack_workspace(T, E, k, d, ffn), dtype=torch.uint8, device="cuda")
    lg = to_dev(np.zeros((2, T, E), np.float32))
    with pytest.raises(mc.MCError):
        mc.stack_forward(x, [s[2] for s in small_stack[:2]], lg, None, TAU, r, x,
                         torch.zeros_like(x), ws)


@pytest.mark.parametrize("T", [1, 64, 1024])
def test_stack_mixtral_two_layers_sampled(mc, T):
    """Mixtral shape (d=4096, ffn=14336, E=8, G=128), two layers of the
    stack, at the benchmark's batches (decode 1 and 64, prefill 1024); sampled tokens (first, last, a protected one), all
    output rows, each layer on the oracle's input rows."""
    c = synthetic.config(5)
    E, d, ffn, G, k = c["E"], c["d"], c["ffn"], c["G"], c["k"]
    x = synthetic.activations(5, T)
    toks = {0, T - 1}
    m0 = synthetic.stack_mask(5, 0, T)
    if m0.any():
        toks.add(int(np.nonzero(m0)[0][0]))
    toks = sorted(toks)
    h = x.copy()
    outs = []
    for l in range(2):
        bits = synthetic.stack_bits(5, l)
        lg = synthetic.stack_logits(5, l, T)
        mask = synthetic.stack_mask(5, l, T)
        rt = oracle.route(lg, mask, k, TAU)
        need = sorted({int(rt["topk_idx"][t, r]) for t in toks for r in range(k) if rt["kept"][t, r]})
        logical = [None] * E
        cache = {}

        def mats(e):
            w = synthetic.stack_expert_weights(5, l, e)
            if e in need:
                cache[e] = w
            return w
        L = pack_layer_gpu(mc, E, d, ffn, bits, G, mats)
        for e in need:
            logical[e] = [oracle.quantize(cache[e][m], bits[e], G) for m in range(3)]
        cache.clear()
        xn = h.copy()
        xn[toks] = oracle.rms_norm(h[toks])
        Y = oracle.moe_forward(xn, rt, logical, G, tokens=toks)
        g = run_stack(mc, h, [L], [lg], [mask], k, E, d, ffn)
        mae, maxrel = check_layer(g[toks], h[toks], Y)
        print("T=%d layer %d tokens %s MAE %.3e MaxRel %.3e" % (T, l, toks, mae, maxrel))
        assert mae <= 1e-3 and maxrel <= 2e-2, (l, mae, maxrel)
        h = h.copy()
        h[toks] = oracle.bf16_round_array(oracle.bf16_to_float64(h[toks]) + Y)
        outs.append(L)
    # the two-layer call equals the chain of the two one-layer calls
    lgs = [synthetic.stack_logits(5, l, T) for l in range(2)]
    masks = [synthetic.stack_mask(5, l, T) for l in range(2)]
    whole = run_stack(mc, x, outs, lgs, masks, k, E, d, ffn)
    step = run_stack(mc, run_stack(mc, x, [outs[0]], [lgs[0]], [masks[0]], k, E, d, ffn),
                     [outs[1]], [lgs[1]], [masks[1]], k, E, d, ffn)
    np.testing.assert_array_equal(whole, step)
