"""GPU parity: the HIP path through the C-ABI against the CPU oracle.

Bit-exact: packed words, scale/zero words, exported codes and fp16
dequantized values, expert selections, kept flags, per-expert lists.
Tolerance (bf16 outputs, fp64 oracle): MAE of |y - bf16(y_ref)| <= 1e-3 and
max |y - y_ref| / max(|y_ref|, rms(y_ref)) <= 2e-2.
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


def u32(t):
    return t.cpu().numpy().view(np.uint32)


def pack_gpu(mc, mats, bits, G, methods=None):
    E = len(mats)
    ffn, d = mats[0][0].shape
    wg = to_dev(np.stack([m[0] for m in mats]))
    wu = to_dev(np.stack([m[1] for m in mats]))
    wd = to_dev(np.stack([m[2] for m in mats]))
    L = mc.PackedLayer(E, d, ffn, bits, G)
    mc.pack(wg, wu, wd, L, methods=methods)
    torch.cuda.synchronize()
    return L


def special_matrices(E, d, ffn, seed=0):
    """Weights with adversarial groups: exact midpoints, constant groups, signed
    zeros, tiny and huge ranges."""
    g = np.random.default_rng(seed)
    mats = []
    for e in range(E):
        per = []
        for shape in ((ffn, d), (ffn, d), (d, ffn)):
            W = (g.standard_normal(shape) * 0.02).astype(np.float32)
            W[0, :32] = 0.25                                   # constant group
            W[1, :32] = np.where(np.arange(32) % 2, 0.0, -0.0)  # signed zeros
            W[2, :32] = np.arange(32) / 31.0 * 0.75            # coarse grid
            W[2, 5] = 0.125
            W[3, :32] = g.standard_normal(32) * 1e-6           # tiny range (s rounds to 0?)
            W[4, :32] = g.standard_normal(32) * 3e4            # huge range (saturating s/z)
            W[5, :32] = np.float32(7.0)
            W[5, 0] = 0.0                                      # min 0, max 7 (ties at x.5)
            W[5, 1:8] = np.array([0.5, 1.5, 2.5, 3.5, 4.5, 5.5, 6.5], np.float32)
            per.append(W)
        mats.append(tuple(per))
    return mats


@pytest.mark.parametrize("case", ["tiny", "special", "olmoe8"])
def test_pack_bit_exact(mc, case):
    if case == "tiny":
        c = synthetic.config(1)
        mats = synthetic.layer_weights(1)
        bits, G = c["bits"], c["G"]
    elif case == "special":
        mats = special_matrices(3, 256, 128)
        bits, G = [1, 2, 3], 32
    else:
        c = synthetic.config(4)
        mats = synthetic.layer_weights(4, E=8)
        bits, G = c["bits"][:8], c["G"]
    words, sz, logical = oracle.pack_layer(mats, bits, G)
    L = pack_gpu(mc, mats, bits, G)
    np.testing.assert_array_equal(u32(L.sz), sz)
    np.testing.assert_array_equal(u32(L.words), words)
    for e in range(len(mats)):
        for m in range(3):
            q, s, z = logical[e][m]
            codes = torch.empty(q.shape, dtype=torch.uint8, device="cuda")
            mc.codes_export(L, e, m, codes)
            deq = torch.empty(q.shape, dtype=torch.float16, device="cuda")
            mc.dequant_export(L, e, m, deq)
            torch.cuda.synchronize()
            np.testing.assert_array_equal(codes.cpu().numpy(), q)
            np.testing.assert_array_equal(deq.cpu().numpy().view(np.uint16),
                                          oracle.dequant_f16(q, s, z, G))


def route_gpu(mc, logits, imp, k, tau):
    T, E = logits.shape
    r = mc.Routing(T, E, k)
    mc.route_and_prune(to_dev(logits), None if imp is None else to_dev(imp), tau, r)
    torch.cuda.synchronize()
    return r


def assert_routing_equal(r, ref, T, k):
    np.testing.assert_array_equal(r.topk_idx.cpu().numpy(), ref["topk_idx"])
    np.testing.assert_array_equal(r.kept.cpu().numpy(), ref["kept"])
    np.testing.assert_array_equal(r.counts.cpu().numpy(), ref["counts"])
    np.testing.assert_array_equal(r.offsets.cpu().numpy(), ref["offsets"])
    n = int(ref["offsets"][-1])
    np.testing.assert_array_equal(r.pair_token.cpu().numpy()[:n], ref["pair_token"][:n])
    np.testing.assert_array_equal(r.pair_rank.cpu().numpy()[:n], ref["pair_rank"][:n])
    np.testing.assert_array_equal(r.pair_pos.cpu().numpy(), ref["pair_pos"])
    assert int(r.n_pruned.cpu()[0]) == ref["n_pruned"]
    np.testing.assert_allclose(r.topk_w.cpu().numpy(), ref["topk_w"], rtol=2e-7, atol=1e-30)
    np.testing.assert_allclose(r.pair_w.cpu().numpy()[:n], ref["pair_w"][:n], rtol=2e-7, atol=1e-30)


def assert_margin(logits, imp, k, tau):
    """For k > 2 the pruning test runs in fp64 on both sides with different exp
    implementations: no normalised weight may sit within 1e-9 of tau."""
    if k <= 2 or tau == 0:
        return
    for t in range(logits.shape[0]):
        l = np.sort(logits[t].astype(np.float64))[::-1][:k]
        p = np.exp(l - l[0])
        p /= p.sum()
        assert np.all(np.abs(p[1:] - tau) > 1e-9 * tau), t


@pytest.mark.parametrize("cid,T,tau", [
    (1, 64, 0.3), (2, 1, 0.3), (2, 8, 0.3), (2, 32, 0.3), (3, 4096, 0.0), (3, 4096, 0.2),
    (3, 4096, 0.4), (4, 2048, 0.05), (4, 16, 0.05), (4, 300, 0.05), (1, 5000, 0.3),
    (2, 65536, 0.3),                                # the token limit: 64 list blocks of 1024
])
def test_route_bit_exact(mc, cid, T, tau):
    c = synthetic.config(cid)
    logits = synthetic.logits(cid, T)
    logits[::5, 1] = logits[::5, 0]                 # exact ties
    imp = synthetic.important_mask(cid, T)
    assert_margin(logits, imp, c["k"], tau)
    ref = oracle.route(logits, imp, c["k"], tau)
    r = route_gpu(mc, logits, imp, c["k"], tau)
    assert_routing_equal(r, ref, T, c["k"])


def test_route_edge_cases(mc):
    g = np.random.default_rng(9)
    # k = 1 (nothing to prune), k = E, E = 256, signed zeros, no mask, tau = 1
    for T, E, k, tau, imp in ((7, 4, 1, 0.3, None), (9, 8, 8, 0.1, None), (33, 256, 8, 0.02, None),
                              (3000, 256, 8, 0.02, None), (1000, 256, 1, 0.3, None),
                              (12, 8, 2, 1.0, None), (12, 8, 2, 0.0, None), (3, 1, 1, 0.5, None)):
        lg = g.standard_normal((T, E)).astype(np.float32)
        lg[0, :] = 0.0
        lg[1, ::2] = -0.0
        assert_margin(lg, imp, k, tau)
        ref = oracle.route(lg, imp, k, tau)
        r = route_gpu(mc, lg, imp, k, tau)
        assert_routing_equal(r, ref, T, k)


@pytest.mark.parametrize("T,E,k,tau", [
    (40, 5, 3, 0.2), (100, 5, 3, 0.2),     # E not a power of two: segments of 8 lanes, k > 2
    (64, 2, 2, 0.3), (200, 2, 2, 0.3),     # 32 tokens per wavefront
    (31, 16, 4, 0.2), (500, 16, 4, 0.2),
    (15, 33, 3, 0.3), (70, 33, 3, 0.3),    # one 64-lane segment, 31 lanes idle
    (48, 16, 4, 0.2), (16, 33, 3, 0.3),    # one launch: one round of the 16 waves (T * E > 512)
])
def test_route_lane_segments(mc, T, E, k, tau):
    """Tokens selected side by side in segments of a wavefront (small batches
    in one launch, larger ones by the selection kernel), with a protection
    mask and ties, against the oracle."""
    g = np.random.default_rng(1000 + T * E)
    lg = g.standard_normal((T, E)).astype(np.float32)
    lg[::3, 1] = lg[::3, 0]
    imp = (g.random(T) < 0.25).astype(np.uint8)
    assert_margin(lg, imp, k, tau)
    ref = oracle.route(lg, imp, k, tau)
    r = route_gpu(mc, lg, imp, k, tau)
    assert_routing_equal(r, ref, T, k)


def layer_case(cid=1, E=None, bits=None, d=None, ffn=None):
    c = synthetic.config(cid)
    E = E or c["E"]
    d = d or c["d"]
    ffn = ffn or c["ffn"]
    bits = bits or c["bits"][:E]
    mats = synthetic.layer_weights(cid, E=E, d=d, ffn=ffn)
    _, _, logical = oracle.pack_layer(mats, bits, c["G"])
    return mats, bits, c["G"], logical


def forward_gpu(mc, L, x_bits, logits, imp, k, tau):
    T, E = logits.shape
    r = route_gpu(mc, logits, imp, k, tau)
    y = torch.empty((T, L.d), dtype=torch.int16, device="cuda")
    ws = torch.empty(mc.forward_workspace(T, E, k, L.d, L.ffn), dtype=torch.uint8, device="cuda")
    mc.moe_forward(to_dev(x_bits.view(np.int16)), r, L, y, ws)
    torch.cuda.synchronize()
    return y.cpu().numpy().view(np.uint16), r


def check_tol(y_bits, y_ref):
    g = oracle.bf16_to_float64(y_bits)
    rb = oracle.bf16_to_float64(oracle.bf16_round_array(y_ref))
    mae = np.abs(g - rb).mean()
    rms = np.sqrt((y_ref ** 2).mean())
    maxrel = (np.abs(g - y_ref) / np.maximum(np.abs(y_ref), rms)).max()
    assert mae <= 1e-3, (mae, maxrel)
    assert maxrel <= 2e-2, (mae, maxrel)
    return mae, maxrel


@pytest.fixture(scope="module")
def tiny(mc):
    mats, bits, G, logical = layer_case(1)
    L = pack_gpu(mc, mats, bits, G)
    return L, logical, G


# T = 4/5 and 8/9: the down and gate/up kernels switch from 8-wave to 16-wave
# workgroups there
@pytest.mark.parametrize("T", [1, 2, 4, 5, 8, 9, 16, 17, 33, 64, 65, 200])
def test_forward_tiny_tolerance(mc, tiny, T):
    L, logical, G = tiny
    x = synthetic.activations(1, T)
    lg = synthetic.logits(1, T)
    imp = synthetic.important_mask(1, T)
    y, _ = forward_gpu(mc, L, x, lg, imp, 2, 0.3)
    ref = oracle.route(lg, imp, 2, 0.3)
    y_ref = oracle.moe_forward(x, ref, logical, G)
    mae, maxrel = check_tol(y, y_ref)
    # the decode and prefill paths dequantize exactly: the error is far below the bar
    assert mae < 2e-4, mae


@pytest.mark.parametrize("d,T", [(640, 1), (768, 5), (1152, 1), (1152, 16), (1152, 17)])
def test_forward_split_reduction(mc, d, T):
    """Batches of at most 16 tokens split the gate/up reduction over d: ragged
    splits (d = 640: 3 + 2 chunks), an empty last split (d = 1152: 3+3+3+0
    chunks) and the unsplit path just above (T = 17)."""
    mats, bits, G, logical = layer_case(1, d=d, ffn=384)
    L = pack_gpu(mc, mats, bits, G)
    x = synthetic.activations(1, T, d=d)
    lg = synthetic.logits(1, T)
    imp = synthetic.important_mask(1, T)
    y, _ = forward_gpu(mc, L, x, lg, imp, 2, 0.3)
    y_ref = oracle.moe_forward(x, oracle.route(lg, imp, 2, 0.3), logical, G)
    mae, _ = check_tol(y, y_ref)
    assert mae < 2e-4, mae


def test_forward_max_tokens_sampled(mc, tiny):
    """The token limit of a call (65536) through the grouped GEMMs: every
    kept pair of the batch is computed, sampled tokens (first, last, a pruned
    one, a protected one, and a seeded spread) are checked against the oracle."""
    L, logical, G = tiny
    T = 65536
    x = synthetic.activations(1, T)
    lg = synthetic.logits(1, T)
    imp = synthetic.important_mask(1, T)
    y, r = forward_gpu(mc, L, x, lg, imp, 2, 0.3)
    ref = oracle.route(lg, imp, 2, 0.3)
    np.testing.assert_array_equal(r.counts.cpu().numpy(), ref["counts"])
    toks = {0, T - 1, int(np.nonzero(ref["kept"][:, 1] == 0)[0][0]), int(np.nonzero(imp)[0][0])}
    toks |= set(np.random.default_rng(65536).choice(T, 60, replace=False).tolist())
    toks = sorted(toks)
    y_ref = oracle.moe_forward(x, ref, logical, G, tokens=toks)
    mae, _ = check_tol(y[toks], y_ref)
    assert mae < 2e-4, mae


@pytest.mark.parametrize("cid,E,d,ffn,T,hot", [
    (1, 4, 256, 512, 300, None),      # G = 32, ragged 32-row fragments
    (1, 4, 384, 256, 257, None),      # d not a multiple of the 256-row down tile
    (1, 4, 256, 512, 600, 1),         # one expert takes every token: 600+ pairs, five 128-token m-tiles
    (4, 16, 2048, 1024, 300, None),   # G = 64, 16 experts, top-8, ragged experts
    (1, 4, 256, 384, 300, None),      # ffn = 384: three 128-row gate/up tiles (ffn % 256 = 128)
    (1, 4, 256, 128, 300, None),      # ffn = 128: a single gate/up row tile
])
def test_forward_prefill_shapes(mc, cid, E, d, ffn, T, hot):
    """Batches above 64 tokens go through the grouped GEMMs: partial 256-token
    tiles (2, 4, 6, 8 fragment rows), experts with no token, G = 32/64/128."""
    c = synthetic.config(cid)
    k = c["k"]
    mats, bits, G, logical = layer_case(cid, E=E, d=d, ffn=ffn)
    L = pack_gpu(mc, mats, bits, G)
    x = synthetic.activations(cid, T, d=d)
    lg = synthetic.logits(cid, T)[:, :E].copy()
    if hot is not None:
        lg[:, hot] += 30.0
    imp = synthetic.important_mask(cid, T)
    tau = c["tau"][0]
    if k > 2:
        assert_margin(lg, imp, k, tau)
    y, r = forward_gpu(mc, L, x, lg, imp, k, tau)
    ref = oracle.route(lg, imp, k, tau)
    y_ref = oracle.moe_forward(x, ref, logical, G)
    mae, maxrel = check_tol(y, y_ref)
    print("prefill cid=%d E=%d d=%d ffn=%d T=%d MAE %.3e MaxRel %.3e" % (cid, E, d, ffn, T, mae, maxrel))


@pytest.mark.parametrize("ffn", [128, 384])
@pytest.mark.parametrize("T", [5, 33])
def test_forward_narrow_ffn_decode(mc, ffn, T):
    """Decode batches with ffn not a multiple of 256 (one or three 128-row
    gate/up blocks)."""
    mats, bits, G, logical = layer_case(1, ffn=ffn)
    L = pack_gpu(mc, mats, bits, G)
    x = synthetic.activations(1, T)
    lg = synthetic.logits(1, T)
    imp = synthetic.important_mask(1, T)
    y, _ = forward_gpu(mc, L, x, lg, imp, 2, 0.3)
    y_ref = oracle.moe_forward(x, oracle.route(lg, imp, 2, 0.3), logical, G)
    mae, _ = check_tol(y, y_ref)
    assert mae < 2e-4, mae


def test_forward_skewed_and_dense(mc, tiny):
    """All tokens on one expert (full token chunks), then tau = 0 with every
    token protected (dense top-k)."""
    L, logical, G = tiny
    T = 64
    x = synthetic.activations(1, T)
    lg = synthetic.logits(1, T)
    lg[:, 2] += 20.0
    for imp, tau in ((None, 0.3), (np.ones(T, np.uint8), 0.0)):
        y, _ = forward_gpu(mc, L, x, lg, imp, 2, tau)
        y_ref = oracle.moe_forward(x, oracle.route(lg, imp, 2, tau), logical, G)
        check_tol(y, y_ref)


def test_forward_single_expert_k1(mc):
    mats, bits, G, logical = layer_case(1, E=1, bits=[3])
    L = pack_gpu(mc, mats, bits, G)
    T = 24
    x = synthetic.activations(1, T)
    lg = np.zeros((T, 1), np.float32)
    y, _ = forward_gpu(mc, L, x, lg, None, 1, 0.3)
    y_ref = oracle.moe_forward(x, oracle.route(lg, None, 1, 0.3), logical, G)
    check_tol(y, y_ref)


def test_forward_olmoe_shaped_small(mc):
    """64 experts, top-8, G = 64, d = 2048 / ffn = 1024 at a reduced expert count
    of the real shape (16 experts) and 16 decode tokens."""
    c = synthetic.config(4)
    E = 16
    mats, bits, G, logical = layer_case(4, E=E)
    L = pack_gpu(mc, mats, bits, G)
    T = 16
    x = synthetic.activations(4, T)
    lg = synthetic.logits(4, T)[:, :E].copy()
    imp = synthetic.important_mask(4, T)
    assert_margin(lg, imp, 8, 0.05)
    y, _ = forward_gpu(mc, L, x, lg, imp, 8, 0.05)
    y_ref = oracle.moe_forward(x, oracle.route(lg, imp, 8, 0.05), logical, G)
    check_tol(y, y_ref)


def test_forward_deterministic(mc, tiny):
    L, logical, G = tiny
    T = 64
    x = synthetic.activations(1, T)
    lg = synthetic.logits(1, T)
    imp = synthetic.important_mask(1, T)
    y1, _ = forward_gpu(mc, L, x, lg, imp, 2, 0.3)
    y2, _ = forward_gpu(mc, L, x, lg, imp, 2, 0.3)
    np.testing.assert_array_equal(y1, y2)


def test_graph_replay_matches_eager(mc, tiny):
    """route_and_prune + moe_forward captured in a HIP graph: every replay, with
    eager work and synchronisations between replays, equals the eager result."""
    L, logical, G = tiny
    T = 32
    x = to_dev(synthetic.activations(1, T).view(np.int16))
    lg = to_dev(synthetic.logits(1, T))
    imp = to_dev(synthetic.important_mask(1, T))
    r = mc.Routing(T, 4, 2)
    y = torch.empty((T, L.d), dtype=torch.int16, device="cuda")
    ws = torch.empty(mc.forward_workspace(T, 4, 2, L.d, L.ffn), dtype=torch.uint8, device="cuda")
    mc.route_and_prune(lg, imp, 0.3, r)
    mc.moe_forward(x, r, L, y, ws)
    torch.cuda.synchronize()
    y_eager = y.clone()
    lists_eager = r.pair_token.clone()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        mc.route_and_prune(lg, imp, 0.3, r)
        mc.moe_forward(x, r, L, y, ws)
    for rep in range(4):
        y.zero_()
        r.pair_token.fill_(-7)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(y, y_eager), rep
        assert torch.equal(r.pair_token[: int(r.offsets[-1])], lists_eager[: int(r.offsets[-1])]), rep
        mc.moe_forward(x, r, L, y, ws)        # eager work between replays
        torch.cuda.synchronize()
        assert torch.equal(y, y_eager)


# ------------------------------------------------------- Eq. 6 importance ---

def importance_gpu(mc, attn_bits, x_bits, rho):
    H, L, _ = attn_bits.shape
    a = to_dev(attn_bits.view(np.int16))
    x = to_dev(x_bits.view(np.int16))
    imp = torch.empty(L, dtype=torch.float32, device="cuda")
    mask = torch.empty(L, dtype=torch.uint8, device="cuda")
    ws = torch.empty(mc.importance_workspace(H, L), dtype=torch.uint8, device="cuda")
    mc.token_importance(a, x, rho, mask, ws, importance=imp)
    torch.cuda.synchronize()
    return imp.cpu().numpy(), mask.cpu().numpy()


def assert_selection_margin(I, n):
    """The n-th and (n+1)-th largest importances differ by more than fp32 noise."""
    if 0 < n < len(I):
        s = np.sort(I)[::-1]
        assert s[n - 1] - s[n] > 1e-5 * s[n - 1], (s[n - 1], s[n])


@pytest.mark.parametrize("H,L,d,rho", [
    (1, 4, 2, 0.5), (2, 300, 64, 0.02), (4, 512, 128, 0.1), (3, 1000, 96, 0.02), (1, 129, 8, 0.5),
    (2, 256, 4096, 0.02), (1, 1, 4, 1.0), (1, 1, 4, 0.4),
])
def test_importance_parity(mc, H, L, d, rho):
    A = synthetic.attention(1, H, L)
    xb = synthetic.activations(1, L, d=d)
    I_ref, m_ref = oracle.token_importance(A, xb, rho)
    assert_selection_margin(I_ref, oracle.protect_count(L, rho))
    I, m = importance_gpu(mc, A, xb, rho)
    np.testing.assert_allclose(I, I_ref, rtol=2e-5, atol=0)
    np.testing.assert_array_equal(m, m_ref)


def test_importance_ties_and_edges(mc):
    """All attention on the first token: every other importance is exactly 0 and
    the remaining protected slots go to the lowest indices; rho = 0 and 1."""
    H, L, d = 2, 200, 32
    A = np.zeros((H, L, L), np.uint16)
    A[:, :, 0] = 0x3F80          # 1.0
    xb = synthetic.activations(1, L, d=d)
    for rho in (0.0, 0.02, 0.1, 1.0):
        I_ref, m_ref = oracle.token_importance(A, xb, rho)
        I, m = importance_gpu(mc, A, xb, rho)
        np.testing.assert_allclose(I, I_ref, rtol=1e-6)
        np.testing.assert_array_equal(m, m_ref)


@pytest.mark.parametrize("H,L,d", [(32, 4096, 4096), (3, 8192, 64)])
def test_importance_large(mc, H, L, d):
    """Mixtral's 32 heads over a 4096-token prefill of d = 4096 (four heads per
    workgroup), and 3 heads over 8192 tokens (head slices of 2 and 1); rho = 2 %."""
    A = synthetic.attention(3, H, L)
    xb = synthetic.activations(3, L, d=d)
    I_ref, m_ref = oracle.token_importance(A, xb, 0.02)
    assert_selection_margin(I_ref, oracle.protect_count(L, 0.02))
    I, m = importance_gpu(mc, A, xb, 0.02)
    np.testing.assert_allclose(I, I_ref, rtol=2e-5)
    np.testing.assert_array_equal(m, m_ref)


# ------------------------------------------------------ sign binarization ---

def _sign_layer(d, ffn):
    mats = synthetic.layer_weights(1, E=4, d=d, ffn=ffn)
    mats[0][0][0, :16] = 0.0
    mats[0][0][1, :16] = -0.0
    mats[0][2][3, :] = np.abs(mats[0][2][3, :])
    return mats, [1, 1, 2, 3], [1, 0, 0, 0]


@pytest.mark.parametrize("d,ffn,G", [(256, 512, 32), (512, 1024, 128)])
def test_pack_sign_binarization_bit_exact(mc, d, ffn, G):
    """Appendix A.2 sign binarization of a 1-bit expert beside RTN experts:
    packed words and scale/zero words bit for bit, exported codes and fp16
    dequantized values."""
    mats, bits, methods = _sign_layer(d, ffn)
    words, sz, logical = oracle.pack_layer(mats, bits, G, methods=methods)
    L = pack_gpu(mc, mats, bits, G, methods)
    assert (u32(L.words) == words).all()
    assert (u32(L.sz) == sz).all()
    for m in range(3):
        q, s, z = logical[0][m]
        R, K = q.shape
        out = torch.empty((R, K), dtype=torch.int16, device="cuda")
        mc.dequant_export(L, 0, m, out)
        torch.cuda.synchronize()
        np.testing.assert_array_equal(out.cpu().numpy().view(np.uint16), oracle.dequant_f16(q, s, z, G).view(np.uint16))


@pytest.mark.parametrize("T", [8, 130])
def test_forward_sign_binarized(mc, T):
    """Forward with a sign-binarized expert (decode and prefill paths)."""
    d, ffn, G = 512, 1024, 128
    mats, bits, methods = _sign_layer(d, ffn)
    _, _, logical = oracle.pack_layer(mats, bits, G, methods=methods)
    L = pack_gpu(mc, mats, bits, G, methods)
    x = synthetic.activations(1, T, d=d)
    lg = synthetic.logits(1, T)
    lg[:, 0] += 1.0                                   # route plenty of tokens to the binarized expert
    imp = synthetic.important_mask(1, T)
    r = mc.Routing(T, 4, 2)
    mc.route_and_prune(to_dev(lg), to_dev(imp), 0.3, r)
    y = torch.empty((T, d), dtype=torch.int16, device="cuda")
    ws = torch.empty(mc.forward_workspace(T, 4, 2, d, ffn), dtype=torch.uint8, device="cuda")
    mc.moe_forward(to_dev(x.view(np.int16)), r, L, y, ws)
    torch.cuda.synchronize()
    ref = oracle.route(lg, imp, 2, 0.3)
    assert ref["counts"][0] > 0
    y_ref = oracle.moe_forward(x, ref, logical, G)
    g = oracle.bf16_to_float64(y.cpu().numpy().view(np.uint16))
    mae = float(np.abs(g - oracle.bf16_to_float64(oracle.bf16_round_array(y_ref))).mean())
    rms = float(np.sqrt((y_ref ** 2).mean()))
    maxrel = float((np.abs(g - y_ref) / np.maximum(np.abs(y_ref), rms)).max())
    assert mae <= 1e-3 and maxrel <= 2e-2, (mae, maxrel)


def test_pack_sign_rejects_wide_expert(mc):
    mats, bits, _ = _sign_layer(256, 512)
    with pytest.raises(mc.MCError):
        pack_gpu(mc, mats, bits, 32, [0, 0, 1, 0])      # expert 2 has 2 bits
