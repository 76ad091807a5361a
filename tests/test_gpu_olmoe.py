"""Parity of the forward at the real OLMoE-shaped layer: d=2048, ffn=1024,
64 experts, top-8, G=64, the workload's widths (iid {1,2,3}), Zipf-skewed
router logits, tau = 0.05 on the normalised top-8 weight (Eq. 1 with k = 8,
Eq. 5 read for k > 2).

Decode (16 tokens) is compared on every output; prefill (2048 tokens, the
grouped GEMMs) on tokens chosen so that every expert holding a token is
covered (experts 16..63 included) together with the first, middle and last
128-token m-tile of the hottest expert, every row."""
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


@pytest.fixture(scope="module")
def olmoe(mc):
    c = synthetic.config(4)
    E, d, ffn, G, bits = c["E"], c["d"], c["ffn"], c["G"], c["bits"]
    assert E == 64 and c["k"] == 8
    mats = synthetic.layer_weights(4)
    L = mc.PackedLayer(E, d, ffn, bits, G)
    wg = to_dev(np.stack([m[0] for m in mats]))
    wu = to_dev(np.stack([m[1] for m in mats]))
    wd = to_dev(np.stack([m[2] for m in mats]))
    mc.pack(wg, wu, wd, L)
    torch.cuda.synchronize()
    del wg, wu, wd
    torch.cuda.empty_cache()
    logical = [[oracle.quantize(mats[e][m], bits[e], G) for m in range(3)] for e in range(E)]
    return c, L, logical


def run(mc, L, c, T):
    E, d, ffn, k, tau = c["E"], c["d"], c["ffn"], c["k"], c["tau"][0]
    x = synthetic.activations(4, T)
    lg = synthetic.logits(4, T)
    imp = synthetic.important_mask(4, T)
    # the k > 2 pruning rule runs in fp64 on both sides: no weight on the boundary
    for t in range(T):
        l = np.sort(lg[t].astype(np.float64))[::-1][:k]
        p = np.exp(l - l[0])
        p /= p.sum()
        assert np.all(np.abs(p[1:] - tau) > 1e-9 * tau), t
    r = mc.Routing(T, E, k)
    mc.route_and_prune(to_dev(lg), to_dev(imp), tau, r)
    y = torch.empty((T, d), dtype=torch.int16, device="cuda")
    ws = torch.empty(mc.forward_workspace(T, E, k, d, ffn), dtype=torch.uint8, device="cuda")
    mc.moe_forward(to_dev(x.view(np.int16)), r, L, y, ws)
    torch.cuda.synchronize()
    ref = oracle.route(lg, imp, k, tau)
    np.testing.assert_array_equal(r.topk_idx.cpu().numpy(), ref["topk_idx"])
    np.testing.assert_array_equal(r.kept.cpu().numpy(), ref["kept"])
    np.testing.assert_array_equal(r.counts.cpu().numpy(), ref["counts"])
    return x, ref, y.cpu().numpy().view(np.uint16)


def check(y_bits, y_ref):
    g = oracle.bf16_to_float64(y_bits)
    rb = oracle.bf16_to_float64(oracle.bf16_round_array(y_ref))
    mae = np.abs(g - rb).mean()
    rms = np.sqrt((y_ref ** 2).mean())
    maxrel = (np.abs(g - y_ref) / np.maximum(np.abs(y_ref), rms)).max()
    assert mae <= 1e-3 and maxrel <= 2e-2, (mae, maxrel)
    return mae, maxrel


def test_olmoe_decode_all_outputs(mc, olmoe):
    c, L, logical = olmoe
    T = 16
    x, ref, y = run(mc, L, c, T)
    touched = np.nonzero(ref["counts"])[0]
    assert (touched >= 16).any()              # experts past the first 16 carry tokens
    y_ref = oracle.moe_forward(x, ref, logical, c["G"])
    mae, maxrel = check(y, y_ref)
    print("OLMoE decode T=16: %d experts touched, MAE %.3e MaxRel %.3e" % (len(touched), mae, maxrel))


def test_olmoe_prefill_every_expert(mc, olmoe):
    c, L, logical = olmoe
    T, k = 2048, c["k"]
    x, ref, y = run(mc, L, c, T)
    counts, offsets, pt = ref["counts"], ref["offsets"], ref["pair_token"]
    toks = {0, T - 1}
    for e in np.nonzero(counts)[0]:           # one token of every expert holding one
        toks.add(int(pt[offsets[e] + counts[e] // 2]))
    hot = int(np.argmax(counts))
    MT = 128                                  # tokens per m-tile of the grouped GEMMs
    n_mt = (int(counts[hot]) + MT - 1) // MT
    assert n_mt >= 3
    for j in (0, n_mt // 2, n_mt - 1):        # first, middle and last m-tile of the hottest expert
        lo = offsets[hot] + MT * j
        hi = min(offsets[hot] + MT * (j + 1), offsets[hot + 1])
        for p in (lo, (lo + hi) // 2, hi - 1):
            toks.add(int(pt[p]))
    toks = sorted(toks)
    covered = {int(e) for t in toks for e, kept in zip(ref["topk_idx"][t], ref["kept"][t]) if kept}
    assert covered == set(np.nonzero(counts)[0].tolist())
    y_ref = oracle.moe_forward(x, ref, logical, c["G"], tokens=toks)
    mae, maxrel = check(y[toks], y_ref)
    print("OLMoE prefill T=2048: %d tokens, %d experts, hot expert %d (%d pairs), MAE %.3e MaxRel %.3e"
          % (len(toks), len(covered), hot, counts[hot], mae, maxrel))
    yall = oracle.bf16_to_float64(y)
    assert np.isfinite(yall).all()
