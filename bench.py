#!/usr/bin/env python3
"""Benchmark of the MC expert path on one MI355X.

Main workload (the paper's Mixtral 8x7b MoE layer shape, synthetic data):
d=4096, ffn=14336, 8 experts, top-2, expert widths [3,3,3,2,2,2,2,3] (2.5 code
bits, the paper's 2.54-bit setting), G=128, decode batch of T tokens (default
32), bf16 activations N(0,1), logits N(0,1) + per-expert bias N(0,0.5^2),
prune threshold 0.3, round(0.1*T) protected tokens.  Also reported in the same
line: decode at 1 and 8 tokens, prefill of 4096 tokens with the threshold
swept over {0, 0.2, 0.4} (pruned fraction, tokens/s, MFMA fraction of the
algorithmic 6*d*ffn FLOPs per kept pair), and the OLMoE-shaped layer (d=2048,
ffn=1024, 64 experts, top-8, G=64, Zipf-skewed logits, threshold 0.05) in
decode (16 tokens) and prefill (2048 tokens), the token importance that
marks the protected tokens (32 heads, 4096 tokens, rho = 0.02), the router
logits ahead of routing, GPTQ of one expert's gate and down matrices, and
the 32-layer residual stack.

One step = route_and_prune + moe_forward over the batch for one layer.  The
step rotates over packed copies of the layer (4 x 484 MB Mixtral, 3 x 131 MB
OLMoE) so the weights come from HBM, not from the 256 MB Infinity Cache.
Prints ONE JSON line.  Per-kernel durations come from the library's HIP-event
instrumentation on the launch stream, recorded over a second pass of the same
timed steps.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, vendor figure
MFMA_PEAK_TFLOPS = 2500.0      # MI355X dense bf16/fp16 MFMA, vendor figure
METRIC = "MoE-layer tokens/s + achieved HBM GB/s (decode) / MFMA % (prefill), 1 GPU"


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=200)
    p.add_argument("--warmup", type=int, default=20)
    p.add_argument("--tokens", type=int, default=32)
    p.add_argument("--copies", type=int, default=4)
    p.add_argument("--sweep", default="1,8", help="extra decode batch sizes to report")
    p.add_argument("--no-cpu", action="store_true", help="skip the oracle baseline")
    p.add_argument("--prefill-steps", type=int, default=10)
    p.add_argument("--no-prefill", action="store_true", help="skip the 4096-token prefill sweep")
    p.add_argument("--no-olmoe", action="store_true", help="skip the OLMoE-shaped layer")
    p.add_argument("--no-importance", action="store_true", help="skip the token-importance measurement")
    p.add_argument("--no-stack", action="store_true", help="skip the 32-layer stack")
    p.add_argument("--no-router", action="store_true", help="skip the router-logits measurement")
    p.add_argument("--no-gptq", action="store_true", help="skip the GPTQ measurement")
    p.add_argument("--stack-steps", type=int, default=10)
    p.add_argument("--no-graph", action="store_true",
                   help="time eager launches only (by default the decode steps are also captured in HIP "
                        "graphs and the replays timed: ms_per_step_graph)")
    p.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                   help="only run a plain device-to-device copy of MIB MiB 5 times (reference "
                        "for the FETCH_SIZE / WRITE_SIZE counters) and exit")
    return p.parse_args()


# Sources of the decode gate/up and down kernels: the stored HBM counter
# figures are reported only while these files are unchanged.
DECODE_SOURCES = ("forward_engine.hpp", "decode.hpp", "mc_device.hpp", "decode_g32.hip", "decode_g64.hip",
                  "decode_g128.hip")


def source_hash() -> str:
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2410_06270_amd", "csrc")
    for name in DECODE_SOURCES:
        with open(os.path.join(csrc, name), "rb") as f:
            h.update(name.encode() + f.read())
    return h.hexdigest()[:16]


def expert_bytes(d, ffn, G, b, mats=(0, 1, 2)):
    """Packed codes + scale/zero words of the listed matrices of one expert."""
    return len(mats) * (d * ffn * b // 8 + d * ffn // G * 4)


class Workload:
    """Packed copies of one synthetic layer (config cid) and a batch of T tokens."""

    def __init__(self, mc, torch, synthetic, T, copies, cid=2):
        c = synthetic.config(cid)
        self.c, self.cid, self.T, self.tau = c, cid, T, c["tau"][0]
        E, d, ffn, k, G, bits = c["E"], c["d"], c["ffn"], c["k"], c["G"], c["bits"]
        self.layers = []
        for cp in range(copies):
            gen = torch.Generator(device="cuda")
            gen.manual_seed(synthetic.BASE_SEED + cid + 1000 * cp)
            w = [torch.randn((E, ffn, d) if m < 2 else (E, d, ffn), generator=gen, device="cuda",
                             dtype=torch.float32).mul_(0.02) for m in range(3)]
            L = mc.PackedLayer(E, d, ffn, bits, G)
            mc.pack(w[0], w[1], w[2], L)
            del w
            self.layers.append(L)
        torch.cuda.synchronize()
        torch.cuda.empty_cache()
        self.set_tokens(mc, torch, synthetic, T)

    def set_tokens(self, mc, torch, synthetic, T, tau=None):
        c, cid = self.c, self.cid
        self.T = T
        self.tau = c["tau"][0] if tau is None else tau
        dev = lambda a: torch.from_numpy(a).cuda()
        self.x = dev(synthetic.activations(cid, T).view("int16"))
        self.logits = dev(synthetic.logits(cid, T))
        self.imp = dev(synthetic.important_mask(cid, T))
        self.r = mc.Routing(T, c["E"], c["k"])
        self.y = torch.empty((T, c["d"]), dtype=torch.int16, device="cuda")
        self.ws = torch.empty(mc.forward_workspace(T, c["E"], c["k"], c["d"], c["ffn"]),
                              dtype=torch.uint8, device="cuda")

    def step(self, mc, i):
        mc.route_and_prune(self.logits, self.imp, self.tau, self.r)
        mc.moe_forward(self.x, self.r, self.layers[i % len(self.layers)], self.y, self.ws)

    def touched(self):
        counts = self.r.counts.cpu().tolist()
        return [e for e, n in enumerate(counts) if n > 0], int(self.r.n_pruned.cpu()[0])

    def kept_pairs(self):
        return int(self.r.offsets.cpu()[-1])

    def alg_bytes(self):
        c = self.c
        d, ffn, G, E = c["d"], c["ffn"], c["G"], c["E"]
        touched, _ = self.touched()
        gateup = sum(expert_bytes(d, ffn, G, c["bits"][e], (0, 1)) for e in touched)
        down = sum(expert_bytes(d, ffn, G, c["bits"][e], (2,)) for e in touched)
        act = self.T * d * 2            # x in (gate/up) and y out (combine)
        logits = self.T * E * 4
        return dict(gateup=gateup + act, down=down, combine=act, step=gateup + down + 2 * act + logits)

    def alg_flops(self):
        """6*d*ffn per kept (token, expert) pair: gate, up (4*d*ffn) and down (2*d*ffn)."""
        P = self.kept_pairs()
        d, ffn = self.c["d"], self.c["ffn"]
        return dict(gateup=4 * d * ffn * P, down=2 * d * ffn * P, step=6 * d * ffn * P)


def time_steps(mc, torch, wl, steps, warmup, graphs=None):
    """Average step time in ms (HIP events around the timed steps).  With
    ``graphs`` (one captured step per layer copy) the steps are graph replays."""
    run = (lambda i: graphs[i % len(graphs)].replay()) if graphs else (lambda i: wl.step(mc, i))
    for i in range(warmup):
        run(i)
    torch.cuda.synchronize()
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    ev0.record()
    for i in range(steps):
        run(i)
    ev1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    return ev0.elapsed_time(ev1) / steps, wall


def capture_steps(mc, torch, wl):
    """One HIP graph per layer copy holding route_and_prune + moe_forward."""
    wl.step(mc, 0)                       # first launches set kernel attributes outside capture
    torch.cuda.synchronize()
    graphs = []
    for cp in range(len(wl.layers)):
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            wl.step(mc, cp)
        graphs.append(g)
    torch.cuda.synchronize()
    return graphs


def kernel_times(mc, torch, wl, steps):
    mc.timing_enable(True)
    for i in range(steps):
        wl.step(mc, i)
    torch.cuda.synchronize()
    out = {}
    for name in ("route_fused", "route_select", "route_lists", "prefill_prep", "gateup", "down", "combine"):
        ms, n = mc.timing_read(name)
        if n:
            out[name] = dict(avg_us=1e3 * ms / n, launches=n)
    mc.timing_enable(False)
    return out


def traffic_from_profiles(kernel, workload, hash_now):
    """HBM bytes per launch measured with rocprofv3 counters (stored summary),
    or None when no summary matches the current kernel sources."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    if not os.path.exists(path):
        return None
    try:
        with open(path) as f:
            rec = json.load(f).get("%s/%s" % (kernel, workload))
    except (OSError, ValueError):
        return None
    if not rec or rec.get("source_hash") != hash_now:
        return None
    return rec.get("bytes_per_launch")


def _cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def _omp_set_threads(n):
    """Thread count of the OpenMP runtime the oracle's C library runs on."""
    import ctypes
    try:
        ctypes.CDLL("libgomp.so.1").omp_set_num_threads(int(n))
        return True
    except (OSError, AttributeError):
        return False


def _random_logical(np, g, E, d, ffn, G, bits, used):
    """Random codes and fp16 scale/zero of the real shapes for the experts in
    ``used`` (the oracle's time does not depend on the values)."""
    logical = []
    for e in range(E):
        if not used[e]:
            logical.append(None)
            continue
        per = []
        for m in range(3):
            R, K = (ffn, d) if m < 2 else (d, ffn)
            q = g.integers(0, 2 ** bits[e], (R, K), dtype=np.uint8)
            s = (np.abs(g.standard_normal((R, K // G))) * 0.01 + 1e-3).astype(np.float16).view(np.uint16)
            z = g.uniform(0, 2 ** bits[e] - 1, (R, K // G)).astype(np.float16).view(np.uint16)
            per.append((q, s, z))
        logical.append(per)
    return logical


def cpu_baseline(synthetic, T, min_seconds=8.0, max_reps=30):
    """The oracle timed on this host, on random codes and fp16 scale/zero of
    the benchmarked shapes (its time does not depend on the values):
      * the headline figure: the full T-token Mixtral-shaped decode batch
        (routing + SwiGLU forward over every kept pair), repeated until at
        least min_seconds of work, with the runtime's default thread count;
      * the same batch restricted to 4 of its tokens on one thread;
      * the 4096-token prefill batch (tau = 0) restricted to a slice of its
        first 256 tokens (every kept pair of those tokens);
      * one layer of the 32-layer stack at T = 1 and T = 64 (the stack's
        per-token rate is the one-layer rate / 32).
    Rates are tokens per second of the sample; the model, nproc and threads
    of the host are reported with them."""
    import numpy as np
    import oracle
    c = synthetic.config(2)
    E, d, ffn, k, G, bits, tau = c["E"], c["d"], c["ffn"], c["k"], c["G"], c["bits"], c["tau"][0]
    threads = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))
    _omp_set_threads(threads)
    g = np.random.default_rng(7)
    logical = _random_logical(np, g, E, d, ffn, G, bits, [True] * E)

    def timed(fn, min_s, reps_max):
        el, reps = 0.0, 0
        while (el < min_s and reps < reps_max) or reps == 0:
            t0 = time.perf_counter()
            fn()
            el += time.perf_counter() - t0
            reps += 1
        return el, reps

    lg, imp, x = synthetic.logits(2, T), synthetic.important_mask(2, T), synthetic.activations(2, T)
    rt = oracle.route(lg, imp, k, tau)
    el, reps = timed(lambda: oracle.moe_forward(x, oracle.route(lg, imp, k, tau), logical, G), min_seconds,
                     max_reps)
    out = dict(value=reps * T / el, unit="tokens/s", cores=threads, kind="oracle",
               seconds=round(el, 3), runs=reps, cpu_model=_cpu_model(), nproc=os.cpu_count(),
               affinity=len(os.sched_getaffinity(0)), threads=threads,
               sample="%d runs of the full T=%d decode batch: routing + SwiGLU forward over its %d kept "
                      "pairs on the d=4096/ffn=14336/E=8 layer (random codes of the same shapes), "
                      "%d OpenMP threads" % (reps, T, int(rt["counts"].sum()), threads))
    # one thread, 4 tokens of the same batch
    if _omp_set_threads(1):
        toks = list(range(4))
        el1, r1 = timed(lambda: oracle.moe_forward(x, rt, logical, G, tokens=toks), 2.0, 5)
        out["single_thread"] = dict(value=round(r1 * len(toks) / el1, 3), unit="tokens/s", threads=1,
                                    seconds=round(el1, 3), sample="%d runs of 4 tokens of the T=%d decode batch"
                                    % (r1, T))
        _omp_set_threads(threads)
    # prefill slice: the first 256 tokens of the 4096-token batch at tau = 0
    c3 = synthetic.config(3)
    lg3, imp3, x3 = synthetic.logits(3, 4096), synthetic.important_mask(3, 4096), synthetic.activations(3, 4096)
    rt3 = oracle.route(lg3, imp3, c3["k"], 0.0)
    toks3 = list(range(256))
    el3, r3 = timed(lambda: oracle.moe_forward(x3, rt3, logical, G, tokens=toks3), 0.0, 1)
    out["prefill_slice"] = dict(value=round(256 * r3 / el3, 3), unit="tokens/s", threads=threads,
                                seconds=round(el3, 3), sample="the first 256 tokens (%d kept pairs) of the "
                                "T=4096 Mixtral-shaped prefill batch, tau = 0"
                                % int(rt3["kept"][:256].sum()))
    # stack slice: one layer at T = 1 and T = 64
    c5 = synthetic.config(5)
    st = {}
    for T5 in (1, 64):
        lg5 = synthetic.stack_logits(5, 0, T5)
        mk5 = synthetic.stack_mask(5, 0, T5)
        x5 = synthetic.activations(5, T5)
        rt5 = oracle.route(lg5, mk5, c5["k"], c5["tau"][0])
        el5, r5 = timed(lambda: oracle.moe_forward(x5, rt5, logical, G), 1.0, 10)
        st["T%d" % T5] = dict(layer_tokens_per_s=round(T5 * r5 / el5, 3),
                              stack_tokens_per_s=round(T5 * r5 / el5 / c5["layers"], 4),
                              seconds=round(el5, 3), runs=r5)
    out["stack_layer_slice"] = dict(st, threads=threads, sample="layer 0 of the 32-layer stack (routing "
                                    "from that layer's logits, expert forward; no RMSNorm/residual), "
                                    "stack rate = layer rate / 32")
    return out


def measure_step(mc, torch, wl, steps, warmup):
    ms, _ = time_steps(mc, torch, wl, steps, warmup)
    kt = kernel_times(mc, torch, wl, steps)
    return ms, {k: v["avg_us"] for k, v in kt.items()}


def prefill_entry(wl, ms, kus):
    fl = wl.alg_flops()
    P, T, k = wl.kept_pairs(), wl.T, wl.c["k"]
    tf = lambda f, us: f / (us * 1e6)       # TFLOP/s
    return dict(tokens=T, tau=wl.tau, pairs_kept=P, pruned_frac=round(1 - P / (T * k), 4),
                tokens_per_s=round(T / (ms / 1e3), 1), ms_per_step=round(ms, 4),
                step_tflops=round(tf(fl["step"], ms * 1e3), 1),
                step_mfma_frac=round(tf(fl["step"], ms * 1e3) / MFMA_PEAK_TFLOPS, 4),
                gateup_mfma_frac=round(tf(fl["gateup"], kus["gateup"]) / MFMA_PEAK_TFLOPS, 4),
                down_mfma_frac=round(tf(fl["down"], kus["down"]) / MFMA_PEAK_TFLOPS, 4),
                kernels_us={k2: round(v, 2) for k2, v in kus.items()})


def decode_entry(wl, ms, kus):
    ab = wl.alg_bytes()
    touched, pruned = wl.touched()
    return dict(tokens=wl.T, tokens_per_s=round(wl.T / (ms / 1e3), 1), ms_per_step=round(ms, 5),
                step_hbm_gbs=round(ab["step"] / (ms * 1e6), 1),
                gateup_hbm_frac=round(ab["gateup"] / (kus["gateup"] * 1e3) / HBM_PEAK_GBS, 4),
                experts_touched=len(touched), pairs_pruned=pruned,
                kernels_us={k2: round(v, 2) for k2, v in kus.items()})


def importance_entry(mc, torch, steps, warmup):
    """Token importance (Eq. 6) + protected set over a 4096-token prefill with
    Mixtral's 32 attention heads and d=4096, rho=0.02.  Inputs drawn on the
    device (torch's generator, seed 20241006): causal row softmaxes of
    N(0, 1.5^2) scores with +4 on the first key, rounded to bf16; x ~ N(0,1)
    in bf16.  The attention map (1.07 GB) exceeds the Infinity Cache, so every
    step reads it from HBM.  Roofline of importance_colsum: the lower triangle
    of bf16 attention, H * L * (L + 1) bytes, plus x (2 * L * d) per launch."""
    H, L, d, rho = 32, 4096, 4096, 0.02
    g = torch.Generator(device="cuda")
    g.manual_seed(20241006)
    attn = torch.empty((H, L, L), dtype=torch.int16, device="cuda")
    above = torch.ones((L, L), dtype=torch.bool, device="cuda").triu_(1)
    for h in range(H):
        sc = torch.randn((L, L), generator=g, device="cuda") * 1.5
        sc[:, 0] += 4.0
        sc.masked_fill_(above, float("-inf"))
        attn[h] = torch.softmax(sc, dim=1).to(torch.bfloat16).view(torch.int16)
        del sc
    x = torch.randn((L, d), generator=g, device="cuda").to(torch.bfloat16).view(torch.int16)
    ws = torch.empty(mc.importance_workspace(H, L), dtype=torch.uint8, device="cuda")
    mask = torch.empty(L, dtype=torch.uint8, device="cuda")
    imp = torch.empty(L, dtype=torch.float32, device="cuda")
    run = lambda: mc.token_importance(attn, x, rho, mask, ws, importance=imp)
    for _ in range(warmup):
        run()
    torch.cuda.synchronize()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ev0.record()
    for _ in range(steps):
        run()
    ev1.record()
    torch.cuda.synchronize()
    ms = ev0.elapsed_time(ev1) / steps
    mc.timing_enable(True)
    for _ in range(steps):
        run()
    torch.cuda.synchronize()
    kus = {}
    for name in ("importance_colsum", "importance_finish", "importance_select"):
        t, n = mc.timing_read(name)
        kus[name] = 1e3 * t / max(n, 1)
    mc.timing_enable(False)
    protected = int(mask.sum().item())
    del attn
    torch.cuda.empty_cache()
    tri = H * L * (L + 1)                        # bytes of the bf16 lower triangle
    colsum_bytes = tri + L * d * 2               # + x, read by the norm workgroups of the same launch
    step_bytes = colsum_bytes + L * 5
    return dict(workload="mixtral_8x7b_token_importance", heads=H, tokens=L, d=d, rho=rho,
                protected=protected, ms_per_step=round(ms, 5), tokens_per_s=round(L / (ms / 1e3), 1),
                step_hbm_gbs=round(step_bytes / (ms * 1e6), 1),
                colsum_alg_bytes=colsum_bytes,
                colsum_hbm_frac=round(colsum_bytes / (kus["importance_colsum"] * 1e3) / HBM_PEAK_GBS, 4),
                kernels_us={k: round(v, 2) for k, v in kus.items()})


def router_entry(mc, torch, synthetic, steps, warmup):
    """Router logits (x W_r^T in fp64 sums, one fp32 rounding) at the Mixtral
    (d=4096, 8 experts) and OLMoE (d=2048, 64 experts) shapes, decode and
    prefill token counts.  x rotates over copies totalling >= 512 MB when one
    copy is large, so prefill-sized x comes from HBM.  Algorithmic bytes per
    launch: x (2*T*d) + W_r (2*E*d) + logits (4*T*E); fp64 work T*E*d
    multiply-adds (peak 78.6 TFLOP/s)."""
    FP64_PEAK_TFLOPS = 78.6
    runs = []
    for cid, T in ((2, 32), (3, 4096), (4, 16), (4, 2048)):
        c = synthetic.config(cid)
        d, E = c["d"], c["E"]
        w = torch.from_numpy(synthetic.router_weights(cid).view("int16")).cuda()
        x0 = torch.from_numpy(synthetic.activations(cid, T).view("int16")).cuda()
        n = max(1, min(64, -(-(512 << 20) // (2 * T * d)))) if 2 * T * d > (8 << 20) else 1
        xs = [x0] + [x0.clone() for _ in range(n - 1)]
        out = torch.empty((T, E), dtype=torch.float32, device="cuda")
        for i in range(warmup):
            mc.router_logits(xs[i % n], w, out)
        torch.cuda.synchronize()
        mc.timing_enable(True)
        for i in range(steps):
            mc.router_logits(xs[i % n], w, out)
        torch.cuda.synchronize()
        t, cnt = mc.timing_read("router")
        mc.timing_enable(False)
        us = 1e3 * t / max(cnt, 1)
        alg = 2 * T * d + 2 * E * d + 4 * T * E
        tflops = 2.0 * T * E * d / (us * 1e-6) / 1e12
        runs.append(dict(workload=c["name"], tokens=T, d=d, experts=E, x_copies=n, kernel_us=round(us, 2),
                         alg_bytes=alg, hbm_gbs=round(alg / (us * 1e3), 1),
                         hbm_frac=round(alg / (us * 1e3) / HBM_PEAK_GBS, 4),
                         fp64_tflops=round(tflops, 2), fp64_frac=round(tflops / FP64_PEAK_TFLOPS, 4)))
        del xs, x0, w, out
        torch.cuda.empty_cache()
    return dict(kernel="router", runs=runs)


def gptq_entry(mc, torch, synthetic):
    """GPTQ (fp64) of one Mixtral expert's gate matrix (14336 x 4096, 3 bits)
    and down matrix (4096 x 14336, 2 bits), G = 128, from 8192 calibration
    rows each, timed per stage with the library's HIP events (one run after
    a warm-up run).  Work per stage: Hessian 2*N*K^2 flops; factor (Cholesky
    and triangular inverse) 4/3*K^3; quantize R*K^2 (one multiply and one
    subtract per compensation term).  Peak: 78.6 fp64 TFLOP/s."""
    FP64_PEAK_TFLOPS = 78.6
    runs = []
    for name, (R, K, bits, tag) in (("gate", (14336, 4096, 3, 1)), ("down", (4096, 14336, 2, 2))):
        N = 8192
        X = torch.from_numpy(synthetic.calibration(2, N, K, tag=tag).view("int16")).cuda()
        W = torch.from_numpy(synthetic.weight(2, 0, 0 if name == "gate" else 2, shape=(R, K))).cuda()
        d, ffn = (K, R) if name == "gate" else (R, K)
        L = mc.PackedLayer(1, d, ffn, [bits], 128)
        H = torch.empty((K, K), dtype=torch.float64, device="cuda")
        U = torch.empty_like(H)
        dead = torch.empty(K, dtype=torch.uint8, device="cuda")
        ws = torch.empty(mc.gptq_workspace(R, K), dtype=torch.uint8, device="cuda")
        mat = 0 if name == "gate" else 2
        def run():
            mc.gptq_hessian(X, H)
            mc.gptq_factor(H, U, dead, ws)
            mc.gptq_quantize(L, 0, mat, W, U, dead, ws)
        run()
        torch.cuda.synchronize()
        mc.timing_enable(True)
        run()
        torch.cuda.synchronize()
        ms = {}
        for st in ("gptq_hessian", "gptq_factor", "gptq_quantize"):
            t, _ = mc.timing_read(st)
            ms[st] = t
        mc.timing_enable(False)
        flops = {"gptq_hessian": 2.0 * N * K * K, "gptq_factor": 4.0 / 3.0 * K ** 3, "gptq_quantize": 1.0 * R * K * K}
        runs.append(dict(matrix=name, rows=R, inputs=K, bits=bits, calib_rows=N,
                         ms={k: round(v, 2) for k, v in ms.items()},
                         fp64_tflops={k: round(flops[k] / (ms[k] * 1e-3) / 1e12, 2) for k in ms},
                         fp64_frac={k: round(flops[k] / (ms[k] * 1e-3) / 1e12 / FP64_PEAK_TFLOPS, 4) for k in ms},
                         total_ms=round(sum(ms.values()), 1)))
        del X, W, L, H, U, dead, ws
        torch.cuda.empty_cache()
    return dict(workload="mixtral_8x7b_expert_gptq", group=128, runs=runs)


def stack_entry(mc, torch, synthetic, steps, warmup, graph=True):
    """The 32-layer Mixtral-shaped expert stack resident in HBM: 32 packed
    layers (widths [3,3,3,2,2,2,2,3] in a seeded order per layer, weights
    N(0, 0.02^2) drawn on the device with a seeded torch generator), each
    layer routed from its own logits (N(0,1) + per-layer expert bias
    N(0, 0.5^2)) with 10 % protected tokens and tau = 0.3, each behind an
    RMSNorm and joined by residual connections (no attention).  One step =
    one mc_moe_stack_forward over all 32 layers; decode batches are also
    captured whole (all 32 layers, one HIP graph) and the replays timed
    (ms_per_step_graph).  Algorithmic bytes: packed
    bytes of every expert a layer routes at least one token to, plus per layer
    the bf16 activations read (norm input, expert input, residual) and written
    (normalised input, output) and the logits."""
    import numpy as np
    c = synthetic.config(5)
    E, d, ffn, k, G, n, tau = c["E"], c["d"], c["ffn"], c["k"], c["G"], c["layers"], c["tau"][0]
    layers, bits = [], []
    for l in range(n):
        gen = torch.Generator(device="cuda")
        gen.manual_seed(synthetic.BASE_SEED + 5 + 1000 * l)
        w = [torch.randn((E, ffn, d) if m < 2 else (E, d, ffn), generator=gen, device="cuda",
                         dtype=torch.float32).mul_(0.02) for m in range(3)]
        b = synthetic.stack_bits(5, l)
        L = mc.PackedLayer(E, d, ffn, b, G)
        mc.pack(w[0], w[1], w[2], L)
        del w
        layers.append(L)
        bits.append(b)
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    resident = sum(L.nbytes for L in layers)
    runs = []
    for T in c["T"]:
        lg = torch.from_numpy(np.stack([synthetic.stack_logits(5, l, T) for l in range(n)])).cuda()
        mk = torch.from_numpy(np.stack([synthetic.stack_mask(5, l, T) for l in range(n)])).cuda()
        x = torch.from_numpy(synthetic.activations(5, T).view("int16")).cuda()
        r = mc.Routing(T, E, k)
        y = torch.empty((T, d), dtype=torch.int16, device="cuda")
        tmp = torch.empty_like(y)
        ws = torch.empty(mc.stack_workspace(T, E, k, d, ffn), dtype=torch.uint8, device="cuda")
        wbytes, kept = 0, 0
        for l in range(n):                      # the library's routing, to count what each layer touches
            mc.route_and_prune(lg[l], mk[l], tau, r)
            counts = r.counts.cpu().tolist()
            wbytes += sum(expert_bytes(d, ffn, G, bits[l][e]) for e in range(E) if counts[e] > 0)
            kept += sum(counts)
        act = n * (5 * T * d * 2 + T * E * 4)
        run = lambda: mc.stack_forward(x, layers, lg, mk, tau, r, y, tmp, ws)
        for _ in range(warmup):
            run()
        torch.cuda.synchronize()
        ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        ev0.record()
        for _ in range(steps):
            run()
        ev1.record()
        torch.cuda.synchronize()
        ms = ev0.elapsed_time(ev1) / steps
        ms_graph = None
        if graph and T <= 64:
            gr = torch.cuda.CUDAGraph()
            with torch.cuda.graph(gr):
                run()
            for _ in range(warmup):
                gr.replay()
            torch.cuda.synchronize()
            ev0.record()
            for _ in range(steps):
                gr.replay()
            ev1.record()
            torch.cuda.synchronize()
            ms_graph = ev0.elapsed_time(ev1) / steps
            del gr
        flops = 6 * d * ffn * kept
        runs.append(dict(tokens=T, path="decode" if T <= 64 else "prefill", ms_per_step=round(ms, 4),
                         ms_per_step_graph=ms_graph and round(ms_graph, 4),
                         tokens_per_s_graph=ms_graph and round(T / (ms_graph / 1e3), 1),
                         tokens_per_s=round(T / (ms / 1e3), 1),
                         alg_bytes=wbytes + act, hbm_gbs=round((wbytes + act) / (ms * 1e6), 1),
                         hbm_frac=round((wbytes + act) / (ms * 1e6) / HBM_PEAK_GBS, 4),
                         pairs_kept=kept, pruned_frac=round(1 - kept / (n * T * k), 4),
                         tflops=round(flops / (ms * 1e9), 1),
                         mfma_frac=round(flops / (ms * 1e9) / MFMA_PEAK_TFLOPS, 4)))
        del lg, mk, x, r, y, tmp, ws
    del layers
    torch.cuda.empty_cache()
    return dict(workload="mixtral_8x7b_moe_stack", layers=n, d=d, ffn=ffn, experts=E, top_k=k,
                group=G, tau=tau, resident_bytes=resident, steps=steps, runs=runs)


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus > 1 or world > 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path "
              "(the sharding design is described in DESIGN.md); run with --gpus 1",
              file=sys.stderr)
        sys.exit(2)
    import torch

    if args.copy_calibration:
        n = args.copy_calibration * (1 << 20) // 4
        src = torch.ones(n, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes": n * 4, "copies": 5}))
        return

    import paper_2410_06270_amd as mc
    import synthetic

    mc.load()
    torch.cuda.set_device(0)
    wl = Workload(mc, torch, synthetic, args.tokens, args.copies)
    c = wl.c
    hash_now = source_hash()

    def measure(T):
        wl.set_tokens(mc, torch, synthetic, T)
        ms, wall = time_steps(mc, torch, wl, args.steps, args.warmup)
        ms_graph = None
        if not args.no_graph:
            ms_graph, _ = time_steps(mc, torch, wl, args.steps, args.warmup, capture_steps(mc, torch, wl))
        kt = kernel_times(mc, torch, wl, args.steps)
        ab = wl.alg_bytes()
        touched, pruned = wl.touched()
        return dict(T=T, ms=ms, ms_graph=ms_graph, wall=wall, kernels=kt, alg=ab, touched=touched,
                    pruned=pruned)

    sweep = []
    for t in [int(v) for v in args.sweep.split(",") if v]:
        if t != args.tokens:
            m = measure(t)
            sweep.append(dict(tokens=t, tokens_per_s=round(t / (m["ms"] / 1e3), 1),
                              ms_per_step=round(m["ms"], 5),
                              ms_per_step_graph=m["ms_graph"] and round(m["ms_graph"], 5),
                              step_hbm_gbs=round(m["alg"]["step"] / (m["ms"] * 1e6), 1),
                              gateup_hbm_frac=round(m["alg"]["gateup"] / (m["kernels"]["gateup"]["avg_us"] * 1e3) / HBM_PEAK_GBS, 4),
                              experts_touched=len(m["touched"])))
    main_m = measure(args.tokens)
    ms_eager = main_m["ms"]
    ms = ms_eager                 # the headline: eager launches (graph replays are reported beside them)
    T = args.tokens
    kt = main_m["kernels"]
    ab = main_m["alg"]
    gu_us = kt["gateup"]["avg_us"]
    achieved = ab["gateup"] / (gu_us * 1e3)        # GB/s
    traffic = traffic_from_profiles("gateup", "mixtral_decode_T%d" % T, hash_now)
    roofline = dict(bound="hbm", kernel="gateup", achieved=round(achieved, 1), peak=HBM_PEAK_GBS,
                    unit="GB/s", frac=round(achieved / HBM_PEAK_GBS, 4), traffic=traffic,
                    alg_bytes_per_launch=ab["gateup"], avg_launch_us=round(gu_us, 3))
    out = {
        "metric": METRIC,
        "value": round(T / (ms / 1e3), 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 5),
        "ms_per_step_graph": main_m["ms_graph"] and round(main_m["ms_graph"], 5),
        "ms_per_step_eager": round(ms_eager, 5),
        "timing": "eager launches of route_and_prune + moe_forward per step, HIP events around the timed "
                  "steps; ms_per_step_graph: the same steps as HIP-graph replays (one graph per layer copy)",
        "kernel_timing": "kernels_us: HIP events around each kernel on its stream in a separate eager pass "
                         "(each figure carries the events' own overhead, about 1-3 us); the roofline's "
                         "avg_launch_us is the gate/up kernel's",
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": "mixtral_8x7b_moe_layer_decode", "d": c["d"], "ffn": c["ffn"],
                   "experts": c["E"], "top_k": c["k"], "bits": c["bits"], "group": c["G"],
                   "tokens": T, "tau": c["tau"][0], "protected": int(synthetic.important_mask(2, T).sum()),
                   "layer_copies": args.copies},
        "step_hbm_gbs": round(ab["step"] / (ms * 1e6), 1),
        "step_hbm_frac": round(ab["step"] / (ms * 1e6) / HBM_PEAK_GBS, 4),
        "experts_touched": len(main_m["touched"]),
        "pairs_pruned": main_m["pruned"],
        "roofline": roofline,
        "kernels_us": {k2: round(v["avg_us"], 3) for k2, v in kt.items()},
        "sweep": sweep,
        "source_hash": hash_now,
    }
    if not args.no_prefill:
        pf = []
        for tau in (0.0, 0.2, 0.4):
            wl.set_tokens(mc, torch, synthetic, 4096, tau)
            ms_p, kus = measure_step(mc, torch, wl, args.prefill_steps, 3)
            pf.append(prefill_entry(wl, ms_p, kus))
        out["prefill"] = {"workload": "mixtral_8x7b_moe_layer_prefill", "tokens": 4096,
                          "mfma_peak_tflops": MFMA_PEAK_TFLOPS, "flops": "6*d*ffn per kept pair",
                          "sweep": pf}
    if not args.no_olmoe:
        del wl
        torch.cuda.empty_cache()
        wo = Workload(mc, torch, synthetic, 16, 3, cid=4)
        ms_d, kus = measure_step(mc, torch, wo, args.steps, args.warmup)
        dec = decode_entry(wo, ms_d, kus)
        wo.set_tokens(mc, torch, synthetic, 2048)
        ms_p, kus = measure_step(mc, torch, wo, args.prefill_steps, 3)
        out["olmoe"] = {"workload": "olmoe_moe_layer", "d": 2048, "ffn": 1024, "experts": 64, "top_k": 8,
                        "group": 64, "bits": wo.c["bits"], "tau": wo.tau, "layer_copies": 3,
                        "decode": dec, "prefill": prefill_entry(wo, ms_p, kus)}
    if not args.no_importance:
        out["importance"] = importance_entry(mc, torch, 20, 3)
    if not args.no_gptq:
        out["gptq"] = gptq_entry(mc, torch, synthetic)
    if not args.no_router:
        out["router"] = router_entry(mc, torch, synthetic, 50, 5)
    if not args.no_stack:
        out["stack"] = stack_entry(mc, torch, synthetic, args.stack_steps, 2, graph=not args.no_graph)
    if not args.no_cpu:
        out["cpu_baseline"] = cpu_baseline(synthetic, T)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
