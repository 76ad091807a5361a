"""mc_moe_forward_noalloc (the forward with the library's own device workspace)
against mc_moe_forward with a caller workspace: identical output bits, on two
calls in a row, the second with a smaller batch (a grouped-GEMM batch of 200
tokens, then an 8-token decode batch), and a request larger than the held
array rejected before any launch."""
import ctypes

import numpy as np
import pytest

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


@pytest.fixture(scope="module")
def mc():
    import paper_2410_06270_amd as m
    m.load()
    return m


def test_noalloc_matches_forward(mc):
    from paper_2410_06270_amd import _binding
    lib = _binding.load()
    E, d, ffn, k, G = 8, 1024, 2048, 2, 128
    bits = [3, 2, 1, 2, 3, 3, 2, 1]
    gen = torch.Generator(device="cuda")
    gen.manual_seed(20241006)
    w = [torch.randn((E, ffn, d) if m < 2 else (E, d, ffn), generator=gen, device="cuda").mul_(0.02)
         for m in range(3)]
    L = mc.PackedLayer(E, d, ffn, bits, G)
    mc.pack(w[0], w[1], w[2], L)
    torch.cuda.synchronize()
    for T in (200, 8):                       # the second call is smaller than the first
        print("noalloc T=%d" % T, flush=True)
        x = (torch.randn((T, d), generator=gen, device="cuda").to(torch.bfloat16)).view(torch.int16)
        lg = torch.randn((T, E), generator=gen, device="cuda")
        imp = (torch.rand((T,), generator=gen, device="cuda") < 0.1).to(torch.uint8)
        r = mc.Routing(T, E, k)
        mc.route_and_prune(lg, imp, 0.3, r)
        y_ref = torch.empty((T, d), dtype=torch.int16, device="cuda")
        ws = torch.empty(mc.forward_workspace(T, E, k, d, ffn), dtype=torch.uint8, device="cuda")
        mc.moe_forward(x, r, L, y_ref, ws)
        y = torch.full((T, d), -1, dtype=torch.int16, device="cuda")
        st = lib.mc_moe_forward_noalloc(x.data_ptr(), ctypes.byref(r.desc), ctypes.byref(L.desc), y.data_ptr(),
                                        ctypes.c_void_p(torch.cuda.current_stream().cuda_stream))
        assert st == 0, lib.mc_last_error()
        torch.cuda.synchronize()
        assert torch.equal(y, y_ref), T
        assert np.isfinite(y.view(torch.bfloat16).float().cpu().numpy()).all()


def test_noalloc_rejects_oversized(mc):
    """A prefill batch whose workspace exceeds the held array: MC_ENOSPACE from
    the host-side check, nothing launched."""
    from paper_2410_06270_amd import _binding
    lib = _binding.load()
    E, d, ffn, k, G, T = 8, 4096, 14336, 2, 128, 4096
    need = mc.forward_workspace(T, E, k, d, ffn)
    assert need > lib_scratch_bytes()
    L = mc.PackedLayer(E, d, ffn, [2] * E, G)
    r = mc.Routing(T, E, k)
    x = torch.zeros((T, d), dtype=torch.int16, device="cuda")
    y = torch.zeros((T, d), dtype=torch.int16, device="cuda")
    st = lib.mc_moe_forward_noalloc(x.data_ptr(), ctypes.byref(r.desc), ctypes.byref(L.desc), y.data_ptr(), None)
    assert st == 2, st                      # MC_ENOSPACE
    assert b"mc_moe_forward_noalloc holds" in lib.mc_last_error()


def lib_scratch_bytes():
    import re
    import os
    hdr = open(os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include",
                            "mc_moe.h")).read()
    m = re.search(r"#define MC_NOALLOC_SCRATCH_BYTES \((\d+)u << (\d+)\)", hdr)
    return int(m.group(1)) << int(m.group(2))
