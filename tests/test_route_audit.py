"""The forward kernels' routing-derived indices stay inside their buffers
for arbitrary routing buffers (CPU audit of the kernels' index helpers).

tests/native/route_audit.hip compiles the helpers of mc_device.hpp that the
decode, combine and prefill kernels use on every index they take from the
routing buffers (expert ranges, pair blocks, token and position clamps, the
prefill set-up's count check) and walks those indices as the kernels do.
Consistent routing from the oracle and garbage buffers (negative, huge and
mutually inconsistent counts, offsets, tokens and positions) must give no
index outside its buffer; the same garbage with the checks bypassed must
(so the garbage does reach past the buffers)."""
import ctypes
import os
import subprocess

import numpy as np
import pytest

import oracle
import synthetic

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "tests", "native", "route_audit.hip")
HDRS = [os.path.join(ROOT, "paper_2410_06270_amd", "csrc", h) for h in ("mc_device.hpp", "prefill.hpp",
                                                                          "forward_engine.hpp")]
LIB = os.path.join(ROOT, "_build", "route_audit.so")


@pytest.fixture(scope="module")
def audit():
    os.makedirs(os.path.dirname(LIB), exist_ok=True)
    if (not os.path.exists(LIB) or os.path.getmtime(LIB) < max(os.path.getmtime(f) for f in [SRC] + HDRS)):
        subprocess.check_call(["hipcc", "--offload-arch=gfx950", "-O1", "-std=c++17", "-shared", "-fPIC",
                               "-o", LIB + ".tmp", SRC])
        os.replace(LIB + ".tmp", LIB)
    lib = ctypes.CDLL(LIB)
    lib.route_audit.restype = ctypes.c_longlong
    mt_tokens = lib.route_audit_mt_tokens()
    p = ctypes.c_void_p

    def run(T, E, k, d, ffn, counts, offsets, pair_token, pair_pos, raw=False):
        arrs = [np.ascontiguousarray(a, dtype=np.int32) for a in (counts, offsets, pair_token, pair_pos)]
        P = T * k
        f_max = (P + 31 * E) // 32          # the prefill workspace's capacities
        mt_max = (P + (mt_tokens - 1) * E) // mt_tokens
        return lib.route_audit(T, E, k, d, ffn, *[p(a.ctypes.data) for a in arrs], f_max, mt_max, int(raw))
    return run


def test_consistent_routing_in_bounds(audit):
    for cid, T in ((1, 64), (2, 32), (3, 4096), (4, 16), (4, 2048)):
        c = synthetic.config(cid)
        r = oracle.route(synthetic.logits(cid, T), synthetic.important_mask(cid, T), c["k"], c["tau"][0])
        assert audit(T, c["E"], c["k"], 256, 512, r["counts"], r["offsets"], r["pair_token"], r["pair_pos"]) == 0


@pytest.mark.parametrize("seed", range(40))
def test_garbage_routing_in_bounds(audit, seed):
    g = np.random.default_rng(seed)
    T = int(g.choice([1, 7, 32, 64, 65, 300]))
    E = int(g.choice([1, 4, 8, 64, 256]))
    k = int(min(E, g.choice([1, 2, 8])))
    P = T * k
    kind = seed % 4
    hi = 1 << 30
    pick = lambda n: np.where(g.random(n) < 0.5, g.integers(-hi, hi, n), g.integers(-2 * P - 2, 2 * P + 2, n))
    counts = pick(E)
    offsets = pick(E + 1)
    if kind == 1:                            # every count at the maximum, offsets all 0
        counts[:] = P
        offsets[:] = 0
    elif kind == 2:                          # counts sum past P, offsets monotone
        counts = g.integers(0, P + 1, E)
        offsets = np.concatenate([[0], np.cumsum(counts)])
    pair_token = pick(P)
    pair_pos = pick(P)
    assert audit(T, E, k, 128, 256, counts, offsets, pair_token, pair_pos) == 0
    if kind == 0:
        # the same buffers without the checks leave the buffers
        assert audit(T, E, k, 128, 256, counts, offsets, pair_token, pair_pos, raw=True) > 0
