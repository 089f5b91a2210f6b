#!/usr/bin/env python3
"""Benchmark of the ring-attention hot path on one MI355X.

Workload (one "step"): causal ring-attention forward, B=1, S=32768, H=32, D=128, bf16
inputs N(0,1), ring of 8 virtual hosts with 4096-token blocks -- partition and ring
schedule, the attention-step kernel on every host (whose workgroups also pass the
key/value block each host holds into the next host's receive buffer), and finalisation.  Inputs are resident in HBM before
the timed region.  Prints ONE JSON line.

  python bench.py [--gpus 1] [--steps K] [--warmup W] [--no-cpu] [--no-extra] [--only NAMES]

`value` is TFLOP/s of algorithmic work (4*B*H*D per visible (query, key) pair; causal
masking halves the diagonal blocks and skips blocks above the diagonal).  The
`roofline` object reports the step kernel's own throughput (HIP events around every
launch, on the stream it runs on, in a second pass of as many calls after the timed ones) against the bf16 dense matrix-core peak, and beside it
against the rates the chip sustains on back-to-back matrix products alone (the library's
calibration kernel, measured in the same run): with fixed operands, and with random
operands that change from product to product as real data does.  `ms_per_step` is the mean over the timed
calls, with their median and minimum alongside.  The
`cpu_baseline` object times the blockwise fp64 ring oracle (torch CPU) on one head of the
same workload and scales it to all 32 heads.  `extra` holds secondary configurations
measured in the same run (forward+backward at S=16384, one host's share at 262144 tokens,
forward and forward+backward, ring decode of 1 and 8 tokens against a 262144-token cache,
blockwise FFN, the Algorithm 1 layer and a 2-layer LLaMA-style training step) for context,
and the same CPU oracle timed on bounded samples of the S=16384 forward+backward and of the
host share.
"""
import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2516.6     # MI355X dense bf16 matrix-core peak (published)
METRIC = "attention fwd / fwd+bwd TFLOPS and % of bf16 MFMA peak; tokens/s at seq 32K-256K"


def causal_pairs(S):
    return S * (S + 1) / 2


def host_pairs(c, host, n_hosts):
    """Visible (query, key) pairs of one host's query block under causal masking."""
    return host * c * c + c * (c + 1) / 2


def time_calls(fn, steps, warmup):
    import torch
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    e0.record()
    for _ in range(steps):
        fn()
    e1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    return e0.elapsed_time(e1) / steps, wall


def time_calls_each(fn, steps):
    """Times `steps` back-to-back calls with an event between consecutive calls: returns
    (mean, median, min) milliseconds per call and the host wall time."""
    import statistics
    import torch
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    t0 = time.perf_counter()
    ev[0].record()
    for i in range(steps):
        fn()
        ev[i + 1].record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    per = [ev[i].elapsed_time(ev[i + 1]) for i in range(steps)]
    return sum(per) / steps, statistics.median(per), min(per), wall


def mfma_loop_peak(ra, torch, random_operands=False, iters=30000, reps=5):
    """Matrix-core throughput the chip sustains with nothing else running (the library's
    calibration kernel: 2048 waves of independent bf16 32x32x16 product chains), TFLOP/s,
    median of `reps` timed launches of ~25-40 ms.  random_operands=False: the same operands
    in every product; True: random operands that change from product to product, as real
    data does (the board then sustains a lower clock)."""
    import statistics
    for _ in range(2):
        ra.mfma_probe(iters, random_operands)
    torch.cuda.synchronize()
    rates = []
    for _ in range(reps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        fl = ra.mfma_probe(iters, random_operands)
        e1.record()
        torch.cuda.synchronize()
        rates.append(fl / (e0.elapsed_time(e1) * 1e-3) / 1e12)
    return statistics.median(rates)


def cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def _torch_threads():
    import torch
    return int(torch.get_num_threads())


def cpu_baseline(B, S, H, D, N):
    """The blockwise ring oracle (fp64, torch CPU) on one head of the workload, scaled to
    all heads."""
    import numpy as np
    from oracle import ring as OR
    rng = np.random.default_rng(0)
    q, k, v = (rng.standard_normal((B, S, 1, D)) for _ in range(3))
    t0 = time.perf_counter()
    OR.ring_attention_fwd(q, k, v, N, True)
    dt = time.perf_counter() - t0
    flops_one_head = 4.0 * B * D * causal_pairs(S)
    return {
        "value": flops_one_head / dt / 1e12,
        "unit": "TFLOP/s",
        "cores": _torch_threads(),
        "cpu_model": cpu_model(),
        "kind": "oracle",
        "sample": "oracle.ring.ring_attention_fwd (blockwise ring oracle, fp64, torch CPU; %d hosts, tiles of "
                  "one block) on 1 of %d heads of the workload (B=%d, S=%d, D=%d, causal): %.1f s; whole "
                  "workload extrapolated linearly to %.0f s" % (N, H, B, S, D, dt, dt * H),
    }


def cpu_baselines_other():
    """The oracle timed on the other configurations: the float32 ring configuration whole
    (S=1024, one head of 64, 4 hosts, forward + backward); forward + backward at S=16384
    (1 of 16 heads); one host's share (host 7 of 8, c=32768; 1 of 32 heads, its first 2 of 8
    ring steps, tiles of 4096); and the Algorithm 1 layer at S=65536, d_model 4096 (its
    forward + backward on 512 rows, scaled linearly in rows for the projections and the
    feed-forward network, plus its attention flops at the S=16384 sample's rate).  Samples
    are extrapolated linearly to the whole configuration."""
    import numpy as np
    from oracle import ring as OR
    rng = np.random.default_rng(1)
    out = {}
    S3, H3, N3, D = 16384, 16, 8, 128
    q, k, v, do = (rng.standard_normal((1, S3, 1, D)) for _ in range(4))
    t0 = time.perf_counter()
    OR.ring_attention_bwd(q, k, v, do, N3, True)  # recomputes the forward: forward + backward
    dt = time.perf_counter() - t0
    f = 4.0 * D * causal_pairs(S3) * 3.5
    out["fwd_bwd_S16384_H16"] = {"tflops": round(f / dt / 1e12, 5), "sample_s": round(dt, 2),
                                 "whole_s_extrapolated": round(dt * H3, 1), "cores": _torch_threads(),
                                 "sample": "1 of 16 heads, ring forward + backward"}
    c5, N5, H5 = 32768, 8, 32
    qb = rng.standard_normal((1, c5, 1, D))
    kk, vv = rng.standard_normal((1, N5 * c5, 1, D)), rng.standard_normal((1, N5 * c5, 1, D))
    t0 = time.perf_counter()
    OR.ring_host_fwd(qb, kk, vv, N5, 7, True, query_chunk=4096, key_chunk=4096, blocks=2)
    dt = time.perf_counter() - t0
    done = c5 * (c5 + 1) / 2 + c5 * c5  # the diagonal block and one full block
    whole = host_pairs(c5, 7, N5) * H5
    out["host7_of_8_c32768_H32"] = {"tflops": round(4.0 * D * done / dt / 1e12, 5), "sample_s": round(dt, 2),
                                    "whole_s_extrapolated": round(dt * whole / done, 1),
                                    "cores": _torch_threads(),
                                    "sample": "1 of 32 heads, the first 2 of 8 ring steps (diagonal + one full block)"}
    S1, N1, D1 = 1024, 4, 64
    q1, k1, v1, do1 = (rng.standard_normal((1, S1, 1, D1)).astype(np.float32) for _ in range(4))
    t0 = time.perf_counter()
    OR.ring_attention_bwd(q1, k1, v1, do1, N1, True)  # forward + backward
    dt = time.perf_counter() - t0
    out["fp32_S1024_H1_D64"] = {"tflops": round(4.0 * D1 * causal_pairs(S1) * 3.5 / dt / 1e12, 5),
                                "sample_s": round(dt, 3), "cores": _torch_threads(),
                                "sample": "the whole configuration, ring forward + backward"}
    from oracle import layer as OL
    S4, Ss, dm, dff, H4 = 65536, 512, 4096, 16384, 32
    x = rng.standard_normal((Ss, dm))
    ws = [rng.standard_normal(sh) * 0.02 for sh in [(dm, dm)] * 4 + [(dm, dff), (dff, dm)]]
    dz = rng.standard_normal((Ss, dm))
    t0 = time.perf_counter()
    OL.layer_fwd(x, *ws, n_heads=H4)
    OL.layer_bwd(x, *ws, dz, n_heads=H4)  # recomputes the forward, as the library does
    dt_rows = time.perf_counter() - t0
    del x, ws, dz
    fatt4 = 4.0 * H4 * D * causal_pairs(S4) * 3.5
    att_rate = out["fwd_bwd_S16384_H16"]["tflops"] * 1e12
    whole = dt_rows * S4 / Ss + fatt4 / att_rate
    flayer = fatt4 + 3 * 24.0 * S4 * dm * dm
    out["layer_fwd_bwd_S65536_d4096"] = {"tflops": round(flayer / whole / 1e12, 5), "sample_s": round(dt_rows, 2),
                                         "whole_s_extrapolated": round(whole, 1), "cores": _torch_threads(),
                                         "sample": "oracle layer forward + backward on 512 rows (projections and "
                                                   "feed-forward network scaled by rows) + attention at the S=16384 "
                                                   "sample's rate"}
    return out


def recorded_traffic():
    """HBM bytes per step-kernel launch from the committed rocprofv3 FETCH_SIZE/WRITE_SIZE
    summary, or None if the kernel sources changed since it was taken."""
    import hashlib
    prof = os.path.join(ROOT, "profiles", "attn_fwd_S32768_H32_D128_hosts8_traffic.md")
    srcs = [os.path.join(ROOT, "paper_2310_01889_amd", "csrc", f)
            for f in ("attn_fwd.hip", "ra_common.h", "ra_kernels.h")]
    if not os.path.exists(prof):
        return None
    h = hashlib.sha256(b"".join(open(f, "rb").read() for f in srcs)).hexdigest()[:16]
    fields = dict(l.split(": ", 1) for l in open(prof).read().splitlines() if ": " in l and not l.startswith("|"))
    if fields.get("source_sha256_16", "").strip() != h:
        return None
    return int(fields["traffic_bytes_per_launch"])


def run_extras(ra, torch, mk, g, D, steps, only):
    """Secondary configurations, each a named section; `only` (a set of names) selects some."""
    extra = {}
    want = lambda name: only is None or name in only

    if want("fwd_bwd"):
        # forward + backward, B=1 S=16384 H=16 D=128, 8 hosts x 2048
        B3, S3, H3, N3 = 1, 16384, 16, 8
        q3, k3, v3, do3 = (mk(B3, S3, H3, D) for _ in range(4))
        o3 = torch.empty_like(q3)
        l3 = torch.empty((B3, H3, S3), dtype=torch.float32, device="cuda")
        dq3, dk3, dv3 = torch.empty_like(q3), torch.empty_like(k3), torch.empty_like(v3)

        def fb():
            ra.ring_attn_fwd(q3, k3, v3, o3, l3, N3, True)
            ra.ring_attn_bwd(q3, k3, v3, o3, l3, do3, dq3, dk3, dv3, N3, True)
        ms3, _ = time_calls(fb, max(3, steps // 2), 2)
        f3 = 4.0 * B3 * H3 * D * causal_pairs(S3) * 3.5
        extra["fwd_bwd_S16384_H16"] = {"ms": round(ms3, 3), "tflops": round(f3 / ms3 / 1e9, 2),
                                       "tokens_per_s": round(S3 / (ms3 * 1e-3), 1)}
        del q3, k3, v3, do3, o3, dq3, dk3, dv3

    c5, N5, H5 = 32768, 8, 32
    if want("host7") or want("decode"):
        k5, v5 = mk(1, N5 * c5, H5, D), mk(1, N5 * c5, H5, D)
    if want("host7"):
        # one host's share: host 7 of 8, 32768-token query block against 262144 keys
        qb = mk(1, c5, H5, D)
        ob = torch.empty_like(qb)
        lb = torch.empty((1, H5, c5), dtype=torch.float32, device="cuda")
        ms5, _ = time_calls(lambda: ra.ring_attn_fwd_host(qb, k5, v5, ob, lb, N5, 7, True), 3, 1)
        f5 = 4.0 * H5 * D * host_pairs(c5, 7, N5)
        extra["host7_of_8_c32768_H32"] = {"ms": round(ms5, 3), "tflops": round(f5 / ms5 / 1e9, 2),
                                          "query_tokens_per_s": round(c5 / (ms5 * 1e-3), 1)}
        # the same share forward + backward: dq local, the float32 dK/dV every block carries
        # received with it through the double buffer, added to and passed on
        dob, dqb = mk(1, c5, H5, D), torch.empty_like(qb)
        dka = torch.zeros((1, N5 * c5, H5, D), dtype=torch.float32, device="cuda")
        dva = torch.zeros_like(dka)

        def fb5():
            ra.ring_attn_fwd_host(qb, k5, v5, ob, lb, N5, 7, True)
            ra.ring_attn_bwd_host(qb, k5, v5, ob, lb, dob, dqb, dka, dva, N5, 7, True)
        for _ in range(2):
            fb5()
        torch.cuda.synchronize()
        ra.timing_read(ra.KERNEL_ATTN_BWD)
        ra.timing_enable(True)
        msb, _ = time_calls(fb5, 3, 0)
        ra.timing_enable(False)
        kb, nb = ra.timing_read(ra.KERNEL_ATTN_BWD)
        ra.timing_read(ra.KERNEL_ATTN_FWD)
        extra["host7_of_8_c32768_H32_fwd_bwd"] = {
            "ms": round(msb, 3), "tflops": round(3.5 * f5 / msb / 1e9, 2),
            "query_tokens_per_s": round(c5 / (msb * 1e-3), 1),
            "bwd_step_kernels_ms": round(kb / 3, 3), "bwd_launches_per_call": nb // 3,
            "bwd_tflops": round(2.5 * f5 / (kb / 3) / 1e9, 2),
            "note": "algorithmic flops: forward + 2.5x for the backward (5 contractions incl. the recompute)"}
        del qb, ob, lb, dob, dqb, dka, dva
    if want("decode"):
        # ring decode against the same 262144-token cache (8 hosts x 32768), 1 and 8 new tokens
        for tq in (1, 8):
            qd = mk(1, tq, H5, D)
            od = torch.empty_like(qd)
            ld = torch.empty((1, H5, tq), dtype=torch.float32, device="cuda")
            dec = lambda: ra.ring_attn_decode(qd, k5, v5, od, ld, N5, True)
            for _ in range(3):
                dec()
            torch.cuda.synchronize()
            ra.timing_read(ra.KERNEL_DECODE)
            ra.timing_enable(True)
            msd, _ = time_calls(dec, 20, 0)
            ra.timing_enable(False)
            kd, nd = ra.timing_read(ra.KERNEL_DECODE)
            kv_bytes = 2.0 * N5 * c5 * H5 * D * 2
            extra["decode_S262144_H32_Tq%d" % tq] = {
                "ms": round(msd, 4), "partial_kernel_ms": round(kd / nd, 4),
                "kv_GBps": round(kv_bytes / (kd / nd) / 1e6, 1),
                "pct_hbm_8TBps": round(100.0 * kv_bytes / (kd / nd) / 1e6 / 8000.0, 1),
                "tokens_per_s": round(tq / (msd * 1e-3), 1)}
    if want("host7") or want("decode"):
        del k5, v5

    # d_model 4096 (32 heads of 128), S = 65536 in 8 host blocks of 8192
    S4, dm, dff, H4, N4 = 65536, 4096, 16384, 32, 8
    w = lambda *shape: (torch.randn(*shape, generator=g, device="cuda") * 0.02).to(torch.bfloat16)
    fatt = 4.0 * H4 * 128 * causal_pairs(S4)
    if want("ffn") or want("layer"):
        x4, dz4 = mk(S4, dm), mk(S4, dm)
        w1, w2 = w(dm, dff), w(dff, dm)
    if want("ffn"):
        # blockwise FFN, d_ff 16384
        y4 = torch.empty_like(x4)
        msf, _ = time_calls(lambda: ra.blockwise_ffn(x4, w1, None, w2, None, y4, S4 // N4), 3, 1)
        fffn = 2.0 * 2 * S4 * dm * dff
        extra["ffn_fwd_T65536_d4096_ff16384"] = {"ms": round(msf, 3), "tflops": round(fffn / msf / 1e9, 2)}
        del y4
    if want("layer"):
        # the Algorithm 1 layer, forward + backward
        wq, wk, wv, wo = (w(dm, dm) for _ in range(4))
        z4, dx4 = torch.empty_like(x4), torch.empty_like(x4)
        f32 = lambda *shape: torch.empty(*shape, dtype=torch.float32, device="cuda")
        dws = [f32(dm, dm) for _ in range(4)] + [f32(dm, dff), f32(dff, dm)]

        def layer():
            ra.ring_layer_fwd(x4, wq, wk, wv, wo, w1, w2, z4, H4, N4, True)
            ra.ring_layer_bwd(x4, wq, wk, wv, wo, w1, w2, dz4, dx4, *dws, H4, N4, True)
        msl, _ = time_calls(layer, 2, 1)
        flayer = 3.5 * fatt + 3 * 24.0 * S4 * dm * dm  # attention fwd+bwd, GEMMs fwd (24 S h^2) + bwd (2x)
        extra["layer_fwd_bwd_S65536_d4096"] = {"ms": round(msl, 3), "tflops": round(flayer / msl / 1e9, 2),
                                               "tokens_per_s": round(S4 / (msl * 1e-3), 1),
                                               "note": "algorithmic flops; backward recomputes the forward"}
        del wq, wk, wv, wo, z4, dx4, dws
    if want("ffn") or want("layer"):
        del x4, dz4, w1, w2
    if want("llama"):
        # training step of a 2-layer LLaMA-7B-width stack (RMSNorm, RoPE, SwiGLU d_ff 11008,
        # pre-norm) around ring attention, full recomputation
        nl, dffl = 2, 11008
        xl, dzl = mk(S4, dm), mk(S4, dm)
        gain = lambda: (1.0 + 0.1 * torch.randn(dm, generator=g, device="cuda")).to(torch.bfloat16)
        params = [[gain(), w(dm, dm), w(dm, dm), w(dm, dm), w(dm, dm), gain(), w(dm, dffl), w(dm, dffl), w(dffl, dm)]
                  for _ in range(nl)]
        grads = [[torch.empty(t.shape, dtype=torch.float32, device="cuda") for t in p] for p in params]
        zl, dxl = torch.empty_like(xl), torch.empty_like(xl)
        msll, _ = time_calls(lambda: ra.llama_stack_train_step(xl, params, dzl, zl, dxl, grads, H4, N4), 2, 1)
        gemm_fwd = 2.0 * S4 * (4 * dm * dm + 3 * dm * dffl)
        fll = nl * (3 * gemm_fwd + 3.5 * fatt)
        extra["llama_stack2_train_step_S65536_d4096_ff11008"] = {
            "ms": round(msll, 2), "tflops": round(fll / msll / 1e9, 2), "tokens_per_s": round(S4 / (msll * 1e-3), 1),
            "note": "algorithmic flops (GEMMs fwd + 2x bwd, attention fwd + 2.5x bwd); the backward recomputes "
                    "each layer's forward"}
    return extra


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    # ~0.4 s of warm-up brings an idle device to its steady clock; 100 timed calls ~0.85 s
    ap.add_argument("--steps", type=int, default=100)
    ap.add_argument("--warmup", type=int, default=50)
    ap.add_argument("--no-cpu", action="store_true", help="skip the CPU oracle baseline")
    ap.add_argument("--no-extra", action="store_true", help="skip the secondary configurations")
    ap.add_argument("--only", default=None,
                    help="comma-separated secondary configurations to run alone (fwd_bwd, host7, decode, ffn, "
                         "layer, llama): no main workload, prints {\"extra\": ...}; for profiling")
    args = ap.parse_args()
    if args.gpus != 1:
        print("bench.py measures one GPU's share of the virtual ring; --gpus %d is not "
              "supported (the ring is emulated on a single device)" % args.gpus, file=sys.stderr)
        sys.exit(2)

    import torch
    import paper_2310_01889_amd as ra

    B, S, H, D, N = 1, 32768, 32, 128, 8
    g = torch.Generator(device="cuda")
    g.manual_seed(2)
    mk = lambda *shape: torch.randn(*shape, generator=g, device="cuda", dtype=torch.float32).to(torch.bfloat16)
    if args.only:
        print(json.dumps({"extra": run_extras(ra, torch, mk, g, D, args.steps, set(args.only.split(",")))}),
              flush=True)
        return
    q, k, v = mk(B, S, H, D), mk(B, S, H, D), mk(B, S, H, D)
    o = torch.empty_like(q)
    lse = torch.empty((B, H, S), dtype=torch.float32, device="cuda")
    step = lambda: ra.ring_attn_fwd(q, k, v, o, lse, N, True)

    flops = 4.0 * B * H * D * causal_pairs(S)
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    # the timed calls run without the library's per-launch timing events (each leaves the
    # GPU idle for a few microseconds between two step kernels); the step kernel's own
    # duration for the roofline is measured in a second pass of as many calls with them
    ms, ms_med, ms_min, wall = time_calls_each(step, args.steps)
    ra.timing_read(ra.KERNEL_ATTN_FWD)
    ra.timing_enable(True)
    for _ in range(args.steps):
        step()
    torch.cuda.synchronize()
    ra.timing_enable(False)
    kms, launches = ra.timing_read(ra.KERNEL_ATTN_FWD)
    k_avg_ms = kms / max(1, launches)
    flops_per_launch = flops / N  # N launches per step
    achieved = flops_per_launch / (k_avg_ms * 1e-3) / 1e12
    value = flops / (ms * 1e-3) / 1e12
    mfma_loop = mfma_loop_peak(ra, torch)
    mfma_loop_rand = mfma_loop_peak(ra, torch, random_operands=True)

    out = {
        "metric": METRIC,
        "value": round(value, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 4),
        "ms_per_step_median": round(ms_med, 4),
        "ms_per_step_min": round(ms_min, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic: N(0,1) bf16 q/k/v drawn on the GPU from a seeded generator",
        "config": {"workload": "causal ring-attention forward, B=1 S=32768 H=32 D=128, "
                               "8 virtual hosts x 4096-token blocks",
                   "global_batch": B, "seq_len": S, "parallelism": "virtual ring of 8 hosts on 1 GPU"},
        "pct_bf16_peak": round(100.0 * value / PEAK_BF16_TFLOPS, 2),
        "tokens_per_s": round(B * S / (ms * 1e-3), 1),
        "roofline": {"bound": "mfma", "kernel": "fwd_bf16_kernel<128, 4> (attention step, four-wave workgroups)",
                     "achieved": round(achieved, 2), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(achieved / PEAK_BF16_TFLOPS, 4), "traffic": recorded_traffic(),
                     "avg_launch_ms": round(k_avg_ms, 4), "launches": launches,
                     "mfma_loop_measured": round(mfma_loop, 1),
                     "frac_of_mfma_loop": round(achieved / mfma_loop, 4),
                     "mfma_loop_random_operands_measured": round(mfma_loop_rand, 1),
                     "frac_of_mfma_loop_random_operands": round(achieved / mfma_loop_rand, 4)},
    }

    if not args.no_extra:
        out["extra"] = run_extras(ra, torch, mk, g, D, args.steps, None)
    if not args.no_cpu:
        out["cpu_baseline"] = cpu_baseline(B, S, H, D, N)
        if not args.no_extra:
            out.setdefault("extra", {})["cpu_oracle_other_configs"] = cpu_baselines_other()
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
