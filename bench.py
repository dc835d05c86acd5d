"""Throughput of OutlierTune's quantized-linear path on one MI355X.

One step = the runtime path of one OPT decoder block's four linears (qkv,
out, fc1, fc2) on the OPT-13B-shaped W6A6 prefill workload (4096 tokens):
for each linear, ot_quantize_act (symmetrize + per-channel quantize) then
ot_qlinear (int8 MFMA GEMM with the fused dequant + bias epilogue).  Inputs
are seeded synthetic activations with structured outlier channels, already
resident in HBM; calibration and the weight fold run once, untimed.

Printed: one JSON line.  `value` is int8 TOPS over the whole step (GEMM ops
2MNK of the four linears divided by the step time, quantization included);
`roofline` covers the dominant kernel (the prefill GEMM) with its duration
measured by HIP events around each launch inside the timed region; the
decode regime (OPT-30B shapes, M in {1, 8, 32, 64}) is reported under
`decode` in GB/s against HBM, on the weights as folded ([N x K]) and on
packed weights (ot_pack_weights, ot_qlinear_packed); `mixed_block` times the paper's own split
(per-channel qkv/fc1, per-token out/fc2); `asym_weights` the main step with
asymmetric ("Int8") weights; `ln_quantize` times the LayerNorm fused with
symmetrization and quantization (qkv and fc1 inputs) against torch's
LayerNorm plus ot_quantize_act; `fp16_baseline` times torch's fp16 linear on
the same shapes; `cpu_baseline` times the CPU oracle on a bounded sample;
`other_prefill` times the OPT-6.7B (W8A8, 2048 tokens) and OPT-66B (W8A8,
8192 tokens) steps the same way, with their fp16 speedup and weight-memory
ratio, and `paper_context` quotes the paper's own speed and memory figures
with the hardware it names.
"""
from __future__ import annotations

import argparse
import concurrent.futures as cf
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = ("ot_qlinear int8 TOPS (%MFMA peak) at OPT-13B prefill; GB/s (%HBM) at decode M≤64")
PEAK_INT8_TOPS = 5000.0    # MI355X dense int8 MFMA, 5.0 POP/s
PEAK_FP16_TFLOPS = 2500.0  # MI355X dense fp16 MFMA
PEAK_HBM_GBS = 8000.0      # MI355X HBM3E, 8 TB/s


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=50)
    p.add_argument("--warmup", type=int, default=10)
    p.add_argument("--workload", default="opt13b_w6a6")
    p.add_argument("--decode-workload", default="opt30b_decode_w8a8")
    p.add_argument("--no-decode", action="store_true", help="skip the decode-regime report")
    p.add_argument("--no-fp16", action="store_true", help="skip the fp16 torch baseline")
    p.add_argument("--no-cpu", action="store_true", help="skip the CPU-oracle baseline")
    p.add_argument("--no-sclk", action="store_true",
                   help="skip the shader-clock window (about 1 s of untimed prefill steps)")
    p.add_argument("--no-ln", action="store_true", help="skip the fused LayerNorm report")
    p.add_argument("--no-other", action="store_true",
                   help="skip the OPT-6.7B and OPT-66B prefill reports")
    p.add_argument("--no-asym", action="store_true",
                   help="skip the asymmetric-weight step report")
    p.add_argument("--no-mixed", action="store_true",
                   help="skip the per-channel + per-token block report")
    p.add_argument("--iters", type=int, default=50, help="iterations for the side measurements")
    p.add_argument("--copy-probe", action="store_true",
                   help="only run a plain 1 GiB device copy (calibrates the HBM byte counters)")
    p.add_argument("--quality", action="store_true",
                   help="only run the symmetrization ablation / bit-width sweep of output error "
                        "against float64 (one JSON line)")
    p.add_argument("--helper-probe", action="store_true",
                   help="launch the quantizer and the fused LayerNorm on the OPT-13B shapes "
                        "(for counter runs)")
    p.add_argument("--helper-traffic", metavar="DIR",
                   help="print the quantizer's and fused LayerNorm's HBM-side traffic from "
                        "counter runs under DIR (host only)")
    p.add_argument("--decode-probe", action="store_true",
                   help="only run each decode-regime linear once per token count (for counter runs)")
    p.add_argument("--counter-summary", metavar="DIR",
                   help="host only: print the markdown summary of the counter runs under DIR "
                        "(mfma/ over the prefill step, dram/ over --decode-probe, dram_copy/ over "
                        "--copy-probe)")
    p.add_argument("--traffic-record", metavar="DIR",
                   help="host only: write the prefill GEMM's HBM traffic record from the "
                        "rocprofv3 counter runs under DIR (fetch/, write/, copy_fetch/, copy_write/)")
    return p.parse_args()


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


# ---------------------------------------------------------------------------
# Workload preparation (untimed): generate, calibrate, fold
# ---------------------------------------------------------------------------
def prepare(wl, rows, torch, ot, synth, pool):
    """Per layer: GPU-resident X (fp16), z, s, inv_s, Wq, sW, b' and the fp16
    weight (kept on the host for the fp16 baseline)."""
    layers = []
    futs = []
    for li, lay in enumerate(wl.layers):
        futs.append((
            pool.submit(synth.weight, wl, li),
            pool.submit(synth.bias, wl, li),
            [pool.submit(synth.activations, wl, li, wl.calib_rows, synth.ROLE_CALIB_X, i)
             for i in range(wl.calib_batches)],
            pool.submit(synth.activations, wl, li, rows),
        ))
    for li, (fw, fb, fcal, fx) in enumerate(futs):
        lay = wl.layers[li]
        batches = (f.result() for f in fcal)
        _, z, s, inv_s = ot.calibrate(batches, wl.a_bits)
        W = torch.from_numpy(fw.result()).cuda()
        b = torch.from_numpy(fb.result()).cuda()
        Wq, sW, bp = ot.fold_weights(W, b, wl.w_bits, z, s)
        X = torch.from_numpy(fx.result()).cuda()
        layers.append(dict(name=lay.name, K=lay.K, N=lay.N, X=X, z=z, s=s, inv_s=inv_s, Wq=Wq,
                           sW=sW, bp=bp, W16=W, b16=b))
        log(f"prepared {wl.name}/{lay.name}: K={lay.K} N={lay.N} rows={rows}")
    return layers


def median_ms(torch, fn, iters, warmup=3):
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(iters)]
    for a, b in ev:
        a.record()
        fn()
        b.record()
    torch.cuda.synchronize()
    t = sorted(a.elapsed_time(b) for a, b in ev)
    return t[len(t) // 2], t[len(t) // 10], t[(9 * len(t)) // 10]


# ---------------------------------------------------------------------------
# Side measurements
# ---------------------------------------------------------------------------
def fp16_baseline(torch, layers, M, iters):
    import torch.nn.functional as F
    def stack():
        for L in layers:
            F.linear(L["X"], L["W16"], L["b16"])
    med, p10, p90 = median_ms(torch, stack, iters)
    ops = sum(2.0 * M * L["N"] * L["K"] for L in layers)
    return dict(ms_per_stack=med, p10_ms=p10, p90_ms=p90, tflops=ops / (med * 1e-3) / 1e12,
                frac_of_fp16_peak=ops / (med * 1e-3) / 1e12 / PEAK_FP16_TFLOPS)


LN_RUN = 10  # fused LayerNorm launches per timed run


def ln_quantize_report(torch, ot, synth, wl, iters):
    """The LayerNorm in front of qkv and fc1 fused with symmetrization and
    quantization (ot_ln_quantize_act), against torch's fp16 LayerNorm
    followed by ot_quantize_act.  Calibration (untimed) runs on torch's fp16
    LayerNorm output of a seeded calibration batch."""
    import torch.nn.functional as F
    out = {}
    for li, lay in enumerate(wl.layers):
        if lay.name not in ("qkv", "fc1"):
            continue
        M, K = wl.M, lay.K
        gamma, beta = (torch.from_numpy(a).cuda() for a in synth.ln_params(wl, li))
        calib = torch.from_numpy(synth.ln_inputs(wl, li, 2048, 1)).cuda()
        _, z, s, inv_s = ot.calibrate([F.layer_norm(calib, (K,), gamma, beta, 1e-5)], wl.a_bits)
        h = torch.from_numpy(synth.ln_inputs(wl, li, M)).cuda()
        Xq = torch.empty((M, K), dtype=torch.int8, device="cuda")
        Xq2 = torch.empty_like(Xq)

        def fused():
            ot.ot_ln_quantize_act(h, gamma, beta, 1e-5, wl.a_bits, z, inv_s, Xq)

        def unfused():
            ot.ot_quantize_act(F.layer_norm(h, (K,), gamma, beta, 1e-5), wl.a_bits, z, inv_s, Xq2)
        # LN_RUN launches back to back per timed run (a ~20 us kernel timed
        # alone carries the events' own overhead), per launch
        def fused_run():
            for _ in range(LN_RUN):
                fused()

        def unfused_run():
            for _ in range(LN_RUN):
                unfused()
        med, p10, p90 = (t / LN_RUN for t in median_ms(torch, fused_run, iters))
        umed = median_ms(torch, unfused_run, iters)[0] / LN_RUN
        nbytes = 3 * M * K + 2 * 2 * K + 2 * 4 * K
        gbs = nbytes / (med * 1e-3) / 1e9
        # the same launch with its input coming from HBM: a 1 GiB buffer is
        # written (untimed) before each launch, which is timed alone
        flush = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
        cold = []
        for _ in range(max(5, iters // 5)):
            flush.fill_(0)
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            fused()
            b.record()
            torch.cuda.synchronize()
            cold.append(a.elapsed_time(b))
        del flush
        cold_ms = float(np.median(cold))
        differ = float((Xq.int() - Xq2.int()).abs().gt(0).float().mean())
        out[lay.name] = dict(M=M, K=K, launches_per_run=LN_RUN, us=med * 1e3, p10_us=p10 * 1e3,
                             p90_us=p90 * 1e3,
                             bytes=nbytes, GBps=gbs, frac_of_hbm_peak=gbs / PEAK_HBM_GBS,
                             input_in_last_level_cache=True,
                             cold_us=cold_ms * 1e3, cold_GBps=nbytes / (cold_ms * 1e-3) / 1e9,
                             cold_note="input evicted from the last-level cache before each "
                                       "launch, launches timed one at a time",
                             unfused_us=umed * 1e3, speedup_vs_unfused=umed / med,
                             codes_differing_from_unfused=differ)
        log(f"ln_quantize {lay.name}: {med * 1e3:.1f} us ({gbs:.0f} GB/s; from HBM "
            f"{cold_ms * 1e3:.1f} us); torch LN + quantize {umed * 1e3:.1f} us")
        del h, calib, Xq, Xq2
    return out


def mixed_block_report(torch, ot, wl, layers, iters):
    """The paper's own split (Sec. 3.2, Sec. 4.1): qkv and fc1 (LayerNorm
    outputs) on the static per-channel path, out and fc2 on the dynamic
    per-token path of Eq. (c).  Same shapes and inputs as the main step;
    the per-token weights are folded (untimed) from the same fp16 weights."""
    M = wl.M
    plan = []
    for L in layers:
        if L["name"] in ("out", "fc2"):
            Wq, sW, bp = ot.fold_weights_per_token(L["W16"], L["b16"], None, wl.w_bits)
            Xq = torch.empty((M, L["K"]), dtype=torch.int8, device="cuda")
            sX = torch.empty(M, dtype=torch.float32, device="cuda")
            plan.append(("token", L, Wq, sW, bp, Xq, sX))
        else:
            plan.append(("channel", L, L["Wq"], L["sW"], L["bp"], L["Xq"], None))

    def step():
        for kind, L, Wq, sW, bp, Xq, sX in plan:
            if kind == "token":
                ot.ot_quantize_act_per_token(L["X"], wl.a_bits, Xq, sX)
                ot.ot_qlinear_per_token(Xq, Wq, sX, sW, bp, wl.a_bits, wl.w_bits, L["Y"])
            else:
                ot.ot_quantize_act(L["X"], wl.a_bits, L["z"], L["inv_s"], Xq)
                ot.ot_qlinear(Xq, Wq, sW, bp, wl.a_bits, wl.w_bits, L["Y"])
    med, p10, p90 = median_ms(torch, step, iters)
    ops = sum(2.0 * M * L["N"] * L["K"] for L in layers)
    # the per-token quantizer alone, on fc2's input
    kind, L, Wq, sW, bp, Xq, sX = plan[3]
    qmed, _, _ = median_ms(torch, lambda: ot.ot_quantize_act_per_token(L["X"], wl.a_bits, Xq, sX),
                           iters)
    qbytes = 3 * M * L["K"] + 4 * M
    log(f"mixed block (per-channel qkv/fc1, per-token out/fc2): {med:.3f} ms "
        f"({ops / (med * 1e-3) / 1e12:.0f} TOPS); per-token quantize fc2 {qmed * 1e3:.1f} us")
    return dict(ms_per_step=med, p10_ms=p10, p90_ms=p90, tops=ops / (med * 1e-3) / 1e12,
                per_token_quantize_fc2_us=qmed * 1e3,
                per_token_quantize_fc2_GBps=qbytes / (qmed * 1e-3) / 1e9)


def asym_report(torch, ot, wl, layers, iters):
    """Asymmetric ("Int8") weights on the main step: the same quantized
    activations against zero-point weight codes (folded untimed from the same
    fp16 weights); the GEMM also forms each token's code sum and subtracts
    zW * sum in the epilogue."""
    M = wl.M
    plan = []
    for L in layers:
        Wq, sW, zW, bp = ot.fold_weights_asym(L["W16"], L["b16"], wl.w_bits, L["z"], L["s"])
        plan.append((L, Wq, sW, zW, bp))

    def step():
        for L, Wq, sW, zW, bp in plan:
            ot.ot_quantize_act(L["X"], wl.a_bits, L["z"], L["inv_s"], L["Xq"])
            ot.ot_qlinear_asym(L["Xq"], Wq, sW, zW, bp, wl.a_bits, wl.w_bits, L["Y"])
    med, p10, p90 = median_ms(torch, step, iters)
    ops = sum(2.0 * M * L["N"] * L["K"] for L in layers)
    log(f"asymmetric-weight step: {med:.3f} ms ({ops / (med * 1e-3) / 1e12:.0f} TOPS)")
    return dict(ms_per_step=med, p10_ms=p10, p90_ms=p90, tops=ops / (med * 1e-3) / 1e12)


DECODE_RUN = 16  # stacks per timed run: a decode loop runs them back to back


def decode_report(torch, ot, synth, wl, pool, iters, with_fp16):
    """Weight-streaming regime: the four linears back to back at M tokens.
    Two copies of the weights alternate so the 256 MB last-level cache cannot
    serve them.  Each timed run is DECODE_RUN stacks back to back, as in a
    decode loop; per-stack figures divide by DECODE_RUN, so the run's one
    launch latency and event overhead are spread over its stacks."""
    Mmax = max(wl.decode_M)
    layers = prepare(wl, Mmax, torch, ot, synth, pool)
    copies = [layers, [dict(L, Wq=L["Wq"].clone(), sW=L["sW"].clone(), bp=L["bp"].clone())
                       for L in layers]]
    packed = [[ot.pack_weights(L["Wq"]) for L in c] for c in copies]
    out = {}
    for M in wl.decode_M:
        xq = [ot.quantize_act(L["X"][:M].contiguous(), wl.a_bits, L["z"], L["inv_s"])
              for L in layers]
        ys = [torch.empty((M, L["N"]), dtype=torch.float16, device="cuda") for L in layers]
        # one scratch buffer serves the stack's calls (they run one after another)
        ws_bytes = max(ot.ot_qlinear_workspace_size(M, L["N"], L["K"]) for L in layers)
        ws = torch.empty(ws_bytes, dtype=torch.uint8, device="cuda") if ws_bytes else None
        wsl = [ws if ot.ot_qlinear_workspace_size(M, L["N"], L["K"]) else None for L in layers]
        it = [0]

        def stack():
            c = copies[it[0] & 1]
            it[0] += 1
            for i, L in enumerate(c):
                ot.ot_qlinear(xq[i], L["Wq"], L["sW"], L["bp"], wl.a_bits, wl.w_bits, ys[i],
                              workspace=wsl[i])

        def run():
            for _ in range(DECODE_RUN):
                stack()
        med, p10, p90 = (t / DECODE_RUN for t in median_ms(torch, run, iters))
        nbytes = sum(L["K"] * L["N"] + M * L["K"] + 2 * M * L["N"] + 8 * L["N"] for L in layers)
        gbs = nbytes / (med * 1e-3) / 1e9
        rec = dict(us_per_stack=med * 1e3, p10_us=p10 * 1e3, p90_us=p90 * 1e3,
                   stacks_per_run=DECODE_RUN, workspace_bytes=ws_bytes,
                   split_k_layers=[L["name"] for L, w in zip(layers, wsl) if w is not None],
                   bytes_per_stack=nbytes, GBps=gbs, frac_of_hbm_peak=gbs / PEAK_HBM_GBS,
                   tokens_per_s=M / (med * 1e-3))
        # the same stack replayed from a HIP graph (what a decode loop does);
        # one graph per weight copy, each replay checked against eager
        ref = [y.clone() for y in ys]
        graphs = []
        for c in copies:
            g = torch.cuda.CUDAGraph()
            torch.cuda.synchronize()
            with torch.cuda.graph(g):
                for i, L in enumerate(c):
                    ot.ot_qlinear(xq[i], L["Wq"], L["sW"], L["bp"], wl.a_bits, wl.w_bits, ys[i],
                                  workspace=wsl[i])
            graphs.append(g)
        for y in ys:
            y.zero_()
        torch.cuda.synchronize()
        for rep in range(3):
            graphs[rep & 1].replay()
            torch.cuda.synchronize()
            assert all(torch.equal(a, b) for a, b in zip(ys, ref)), "graph replay differs"
        gi = [0]

        def replay():
            for _ in range(DECODE_RUN):
                graphs[gi[0] & 1].replay()
                gi[0] += 1
        gmed = median_ms(torch, replay, iters)[0] / DECODE_RUN
        rec["graph_us_per_stack"] = gmed * 1e3
        rec["graph_GBps"] = nbytes / (gmed * 1e-3) / 1e9
        rec["graph_frac_of_hbm_peak"] = rec["graph_GBps"] / PEAK_HBM_GBS
        del graphs
        # the same stack on packed weights (ot_pack_weights, untimed, like the
        # fold), checked bit for bit against the standard layout's outputs
        yp = [torch.empty_like(y) for y in ys]
        itp = [0]

        def stack_packed():
            c = packed[itp[0] & 1]
            itp[0] += 1
            for i, L in enumerate(layers):
                ot.ot_qlinear_packed(xq[i], c[i], L["N"], L["sW"], L["bp"], wl.a_bits,
                                     wl.w_bits, yp[i], workspace=wsl[i])

        def run_packed():
            for _ in range(DECODE_RUN):
                stack_packed()
        for c in copies:  # one eager stack per copy on the standard layout, for the check
            for i, L in enumerate(c):
                ot.ot_qlinear(xq[i], L["Wq"], L["sW"], L["bp"], wl.a_bits, wl.w_bits, ys[i],
                              workspace=wsl[i])
        stack_packed()
        stack_packed()
        torch.cuda.synchronize()
        assert all(torch.equal(a, b) for a, b in zip(yp, ys)), "packed outputs differ"
        pmed, pp10, pp90 = (t / DECODE_RUN for t in median_ms(torch, run_packed, iters))
        rec["packed_us_per_stack"] = pmed * 1e3
        rec["packed_p10_us"], rec["packed_p90_us"] = pp10 * 1e3, pp90 * 1e3
        rec["packed_GBps"] = nbytes / (pmed * 1e-3) / 1e9
        rec["packed_frac_of_hbm_peak"] = rec["packed_GBps"] / PEAK_HBM_GBS
        rec["packed_tokens_per_s"] = M / (pmed * 1e-3)
        if with_fp16:
            import torch.nn.functional as F
            w16 = [[L["W16"] for L in layers], [L["W16"].clone() for L in layers]]
            x16 = [L["X"][:M].contiguous() for L in layers]
            it16 = [0]

            def stack16():
                for _ in range(DECODE_RUN):
                    ws = w16[it16[0] & 1]
                    it16[0] += 1
                    for i, L in enumerate(layers):
                        F.linear(x16[i], ws[i], L["b16"])
            m16 = median_ms(torch, stack16, iters)[0] / DECODE_RUN
            rec["fp16_us_per_stack"] = m16 * 1e3
            rec["speedup_vs_fp16"] = m16 / med
            del w16
        out[str(M)] = rec
        log(f"decode M={M}: {med * 1e3:.1f} us/stack, {gbs:.0f} GB/s; graph "
            f"{gmed * 1e3:.1f} us, {rec['graph_GBps']:.0f} GB/s; packed weights "
            f"{pmed * 1e3:.1f} us, {rec['packed_GBps']:.0f} GB/s")
    return out


TRAFFIC_RECORD = os.path.join(ROOT, "profiles", "qgemm_prefill_opt13b_w6a6_traffic.json")
PREFILL_SOURCES = [os.path.join(ROOT, "paper_2406_18832_amd", "csrc", f)
                   for f in ("ot_prefill.hip", "ot_gemm_common.h")]


def prefill_source_digest():
    import hashlib
    h = hashlib.sha256()
    for path in PREFILL_SOURCES:
        with open(path, "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def measured_traffic():
    """HBM bytes per prefill-GEMM launch from the committed counter summary,
    if it was taken on the current prefill kernel source; else None."""
    try:
        with open(TRAFFIC_RECORD) as f:
            rec = json.load(f)
        digest = prefill_source_digest()
    except OSError:
        return None
    if rec.get("source_sha256") != digest:
        return None
    return rec.get("traffic_bytes_per_launch")


def _counter_rows(d, counter):
    import csv
    import glob
    rows = []
    for path in sorted(glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True)):
        with open(path) as f:
            rows += [r for r in csv.DictReader(f) if r["Counter_Name"] == counter]
    if not rows:
        raise SystemExit(f"no {counter} rows under {d}")
    return rows


def _per_dispatch(rows, name_part):
    """Counter value summed per dispatch (in dispatch order) for kernels whose
    name contains name_part, with each dispatch's grid size."""
    acc, grid = {}, {}
    for r in rows:
        if name_part not in r["Kernel_Name"]:
            continue
        d = int(r["Dispatch_Id"])
        acc[d] = acc.get(d, 0.0) + float(r["Counter_Value"])
        grid[d] = int(r["Grid_Size"])
    return [(grid[d], acc[d]) for d in sorted(acc)]


def prefill_fetch_floor(M, N, K, bn, bm, group_m=8, xcds=8, per_xcd=32):
    """Least HBM-side operand fetch (bytes) of one prefill launch under the
    kernel's tile schedule: the workgroups are dealt to the XCDs in
    contiguous ranges and walked in groups of group_m token tiles, and each
    XCD runs per_xcd of them at a time (one per CU); its L2 can share the
    operand panels only among those, so per XCD and pass every distinct
    token panel (bm rows) and channel panel (bn rows) is fetched over all of
    K once."""
    tiles_m, tiles_n = -(-M // bm), -(-N // bn)
    nwg = tiles_m * tiles_n
    per, rem = nwg // xcds, nwg % xcds
    total = 0
    for x in range(xcds):
        n_x = per + (1 if x < rem else 0)
        start = x * (per + 1) if x < rem else rem * (per + 1) + (x - rem) * per
        for p0 in range(start, start + n_x, per_xcd):
            tms, tns = set(), set()
            for lid in range(p0, min(p0 + per_xcd, start + n_x)):
                gs = group_m * tiles_n
                first_m = (lid // gs) * group_m
                gm = min(tiles_m - first_m, group_m)
                tms.add(first_m + (lid % gs) % gm)
                tns.add((lid % gs) // gm)
            total += (len(tms) * bm + len(tns) * bn) * K
    return total


def traffic_record(d, workload):
    """Writes the prefill GEMM's HBM traffic record from four rocprofv3 --pmc
    runs under d: fetch/ and write/ (FETCH_SIZE, WRITE_SIZE of `bench.py
    --steps 2 --warmup 1 --no-cpu --no-fp16 --no-decode`), copy_fetch/ and
    copy_write/ (the same counters over `bench.py --copy-probe`).  Host only."""
    from paper_2406_18832_amd import synth
    wl = synth.WORKLOADS[workload]
    n_copy = 1 << 30  # bytes read and written per copy_probe launch
    factors = {}
    for c, sub in (("FETCH_SIZE", "copy_fetch"), ("WRITE_SIZE", "copy_write")):
        disp = _per_dispatch(_counter_rows(os.path.join(d, sub), c), "copyBuffer")
        kib = [v for _, v in disp if v > 0.5 * n_copy / 1024 / 4]
        factors[c] = n_copy / 1024 / float(np.median(kib))
    per = {L.name: {"fetch_kib": [], "write_kib": []} for L in wl.layers}
    tile_of = {}
    threads = 512  # workgroup size of the prefill kernel (8 waves)
    for c, sub, key in (("FETCH_SIZE", "fetch", "fetch_kib"), ("WRITE_SIZE", "write", "write_kib")):
        disp = _per_dispatch(_counter_rows(os.path.join(d, sub), c), "qgemm_prefill_kernel")
        if len(disp) % len(wl.layers):
            raise SystemExit(f"{len(disp)} prefill dispatches is not a whole number of steps")
        for i, (g, v) in enumerate(disp):
            L = wl.layers[i % len(wl.layers)]
            # the library runs 256 x 256, 320 (channels) x 256 (tokens), 256 x 128 or
            # 192 x 256 tiles
            grids = {f"{bn}x{bm}": -(-wl.M // bm) * -(-L.N // bn) * threads
                     for bn, bm in ((256, 256), (320, 256), (256, 128), (192, 256))}
            match = [t for t, gg in grids.items() if gg == g]
            if not match:
                raise SystemExit(f"dispatch {i}: grid {g} fits no tile shape of layer {L.name} "
                                 f"({grids})")
            tile_of[L.name] = match[0]
            per[L.name][key].append(v)
    rec_layers, alg = {}, {}
    for L in wl.layers:
        f = float(np.mean(per[L.name]["fetch_kib"]))
        w = float(np.mean(per[L.name]["write_kib"]))
        bn, bm = (int(v) for v in tile_of[L.name].split("x"))
        rec_layers[L.name] = {"fetch_kib": f, "write_kib": w, "tile": tile_of[L.name],
                              "bytes": (f * factors["FETCH_SIZE"] + w * factors["WRITE_SIZE"]) * 1024,
                              "fetch_floor_bytes": prefill_fetch_floor(wl.M, L.N, L.K, bn, bm)}
        alg[L.name] = wl.M * L.K + L.N * L.K + 2 * wl.M * L.N + 8 * L.N
    cmd = "cd /tmp && timeout -s KILL 120 rocprofv3 --pmc {c} --output-format csv -d <out>/{sub} -o p -- python -u <repo>/bench.py {args}"
    bench_args = ("--steps 2 --warmup 1 --no-cpu --no-fp16 --no-decode --no-ln --no-mixed "
                  "--no-asym --no-sclk --no-other")
    rec = {
        "kernel": "qgemm_prefill_kernel (256x256, 320x256, 256x128 or 192x256 tiles, BK 128, 2 stages)",
        "workload": f"{wl.name} ({wl.M} tokens; " + ", ".join(L.name for L in wl.layers) + ")",
        "source_files": [os.path.relpath(p, ROOT) for p in PREFILL_SOURCES],
        "source_sha256": prefill_source_digest(),
        "copy_factor_fetch": factors["FETCH_SIZE"],
        "copy_factor_write": factors["WRITE_SIZE"],
        "per_layer": rec_layers,
        "algorithmic_bytes_per_layer": alg,
        "traffic_bytes_per_launch": float(np.mean([v["bytes"] for v in rec_layers.values()])),
        "algorithmic_bytes_per_launch": float(np.mean(list(alg.values()))),
        "commands": [cmd.format(c="FETCH_SIZE", sub="fetch", args=bench_args),
                     cmd.format(c="WRITE_SIZE", sub="write", args=bench_args),
                     cmd.format(c="FETCH_SIZE", sub="copy_fetch", args="--copy-probe"),
                     cmd.format(c="WRITE_SIZE", sub="copy_write", args="--copy-probe"),
                     f"python bench.py --traffic-record <out>"],
    }
    with open(TRAFFIC_RECORD, "w") as f:
        json.dump(rec, f, indent=1)
    print(json.dumps({k: rec[k] for k in ("traffic_bytes_per_launch", "algorithmic_bytes_per_launch",
                                          "copy_factor_fetch", "copy_factor_write")}))


def decode_probe(torch, ot, synth, wl, pool):
    """Each decode-regime linear once per token count, in a fixed order
    (row-major weights, then packed; M ascending; qkv, out, fc1, fc2), as
    the bench runs it (workspace where the library uses one); for counter
    runs."""
    layers = prepare(wl, max(wl.decode_M), torch, ot, synth, pool)
    for L in layers:
        L["Wp"] = ot.pack_weights(L["Wq"])
    plan = []
    for packed in (False, True):
        for M in wl.decode_M:
            for L in layers:
                xq = ot.quantize_act(L["X"][:M].contiguous(), wl.a_bits, L["z"], L["inv_s"])
                y = torch.empty((M, L["N"]), dtype=torch.float16, device="cuda")
                plan.append((packed, M, L, xq, y, ot.workspace_for(M, L["N"], L["K"])))
    torch.cuda.synchronize()
    for packed, M, L, xq, y, ws in plan:
        if packed:
            ot.ot_qlinear_packed(xq, L["Wp"], L["N"], L["sW"], L["bp"], wl.a_bits, wl.w_bits, y,
                                 workspace=ws)
        else:
            ot.ot_qlinear(xq, L["Wq"], L["sW"], L["bp"], wl.a_bits, wl.w_bits, y, workspace=ws)
    torch.cuda.synchronize()
    print(json.dumps({"decode_probe": [[p, M, L["name"], ws is not None]
                                       for p, M, L, _, _, ws in plan]}))


def counter_summary(d, workload, decode_workload):
    """Markdown summary of three rocprofv3 --pmc runs under d (host only):
    mfma/ (SQ_INSTS_VALU_MFMA_MOPS_I8, SQ_VALU_MFMA_BUSY_CYCLES,
    SQ_BUSY_CU_CYCLES, GRBM_GUI_ACTIVE, SQ_LDS_BANK_CONFLICT, SQ_INSTS_LDS
    over the prefill step), dram/ (TCC_EA0_RDREQ_DRAM_32B,
    TCC_EA0_WRREQ_WRITE_DRAM_32B over --decode-probe), dram_copy/ (the
    same over --copy-probe) and, if present, dram_prefill/ (the same over
    the prefill step).  rocprofv3 sums each counter over its hardware
    instances; GRBM_GUI_ACTIVE is counted once per XCD, so it is divided by
    the 8 XCDs."""
    import csv
    import glob
    from paper_2406_18832_amd import synth

    def dispatches(sub):
        rows = []
        for path in sorted(glob.glob(os.path.join(d, sub, "**", "*counter_collection.csv"),
                                     recursive=True)):
            with open(path) as f:
                rows += list(csv.DictReader(f))
        by = {}
        for r in rows:
            e = by.setdefault(int(r["Dispatch_Id"]), {"name": r["Kernel_Name"],
                                                      "grid": int(r["Grid_Size"]),
                                                      "ns": int(r["End_Timestamp"])
                                                      - int(r["Start_Timestamp"])})
            e[r["Counter_Name"]] = e.get(r["Counter_Name"], 0.0) + float(r["Counter_Value"])
        return [by[k] for k in sorted(by)]

    simds, xcds = 1024, 8
    wl = synth.WORKLOADS[workload]
    pre = [e for e in dispatches("mfma") if "qgemm_prefill_kernel" in e["name"]]
    out = ["| Layer | Tile | int8 ops counted (MOPS_I8 x 512) | 2MNK | MFMA busy / (GUI active x 1024 SIMDs) | LDS bank-conflict cycles / LDS instr | shader clock: GUI active per XCD / dispatch time |",
           "|---|---|---|---|---|---|---|"]
    for i, L in enumerate(wl.layers):
        es = pre[i::len(wl.layers)]
        ops = np.mean([e["SQ_INSTS_VALU_MFMA_MOPS_I8"] * 512 for e in es])
        util = np.mean([e["SQ_VALU_MFMA_BUSY_CYCLES"] / (e["GRBM_GUI_ACTIVE"] / xcds * simds)
                        for e in es])
        confl = np.mean([e["SQ_LDS_BANK_CONFLICT"] / max(e["SQ_INSTS_LDS"], 1) for e in es])
        ghz = np.mean([e["GRBM_GUI_ACTIVE"] / xcds / e["ns"] for e in es])
        tile = "?"
        for bn, bm in ((256, 256), (320, 256), (256, 128), (192, 256)):
            if es[0]["grid"] == -(-wl.M // bm) * -(-L.N // bn) * 512:
                tile = f"{bn}x{bm}"
        out.append(f"| {L.name} | {tile} | {ops:.4g} | {2 * wl.M * L.N * L.K:.4g} | {util:.3f} | "
                   f"{confl:.3f} | {ghz:.2f} GHz |")
    copy = [e for e in dispatches("dram_copy") if "copyBuffer" in e["name"]]
    n_copy = 1 << 30
    big = [e for e in copy if e["TCC_EA0_RDREQ_DRAM_32B"] * 32 > n_copy / 4]
    rd_f = n_copy / float(np.median([e["TCC_EA0_RDREQ_DRAM_32B"] * 32 for e in big]))
    wr_f = n_copy / float(np.median([e["TCC_EA0_WRREQ_WRITE_DRAM_32B"] * 32 for e in big]))
    dwl = synth.WORKLOADS[decode_workload]
    dec = [e for e in dispatches("dram") if "qgemm_decode" in e["name"] or "decode_reduce" in e["name"]]
    order = [(p, M, L) for p in ("row-major", "packed") for M in dwl.decode_M
             for L in dwl.layers]
    out2 = ["| Weights | M | Layer | kernels | DRAM read bytes | DRAM write bytes | algorithmic bytes | read / algorithmic |",
            "|---|---|---|---|---|---|---|---|"]
    i = 0
    for p, M, L in order:
        ks = [dec[i]]
        i += 1
        if "split" in ks[0]["name"]:
            ks.append(dec[i])
            i += 1
        rd = sum(e["TCC_EA0_RDREQ_DRAM_32B"] for e in ks) * 32 * rd_f
        wr = sum(e["TCC_EA0_WRREQ_WRITE_DRAM_32B"] for e in ks) * 32 * wr_f
        alg = L.K * L.N + M * L.K + 2 * M * L.N + 8 * L.N
        out2.append(f"| {p} | {M} | {L.name} | {len(ks)} | {rd / 1e6:.1f} MB | {wr / 1e6:.2f} MB | "
                    f"{alg / 1e6:.1f} MB | {rd / alg:.3f} |")
    if i != len(dec):
        raise SystemExit(f"{len(dec)} decode dispatches, {i} accounted for")
    out3 = []
    if os.path.isdir(os.path.join(d, "dram_prefill")):
        pre_d = [e for e in dispatches("dram_prefill") if "qgemm_prefill_kernel" in e["name"]]
        out3 = ["| Layer | DRAM read bytes | DRAM write bytes | algorithmic reads (Xq + Wq + sW + b') | reads / algorithmic |",
                "|---|---|---|---|---|"]
        for li, L in enumerate(wl.layers):
            es = pre_d[li::len(wl.layers)]
            rd = np.mean([e["TCC_EA0_RDREQ_DRAM_32B"] for e in es]) * 32 * rd_f
            wr = np.mean([e["TCC_EA0_WRREQ_WRITE_DRAM_32B"] for e in es]) * 32 * wr_f
            alg = wl.M * L.K + L.N * L.K + 8 * L.N
            out3.append(f"| {L.name} | {rd / 1e6:.1f} MB | {wr / 1e6:.1f} MB | {alg / 1e6:.1f} MB | "
                        f"{rd / alg:.3f} |")
    out4 = []
    if os.path.isdir(os.path.join(d, "diag")):
        # what the K loop waits on: L1-to-L2 read latency, L2 hit rate and
        # the vector memory pipeline's busy and stall cycles, per CU per
        # active cycle
        pre_g = [e for e in dispatches("diag") if "qgemm_prefill_kernel" in e["name"]]
        cus = 256
        out4 = ["| Layer | L1-to-L2 read latency (cycles per request) | L2 hit rate | TA busy | TA address stalled by TC | TCP stalled on pending L2 data |",
                "|---|---|---|---|---|---|"]
        for li, L in enumerate(wl.layers):
            es = pre_g[li::len(wl.layers)]

            def per_cu(key):
                return np.mean([e[key] / (e["GRBM_GUI_ACTIVE"] / xcds) / cus for e in es])
            lat = np.mean([e["TCP_TCC_READ_REQ_LATENCY"] / e["TCP_TCC_READ_REQ"] for e in es])
            hit = np.mean([e["TCC_HIT"] / (e["TCC_HIT"] + e["TCC_MISS"]) for e in es])
            out4.append(f"| {L.name} | {lat:.0f} | {hit:.3f} | {per_cu('TA_TA_BUSY'):.2f} | "
                        f"{per_cu('TA_ADDR_STALLED_BY_TC_CYCLES'):.2f} | "
                        f"{per_cu('TCP_PENDING_STALL_CYCLES'):.2f} |")
    print("\n".join(out))
    print()
    print(f"DRAM counter calibration on a 1 GiB copy: read factor {rd_f:.3f}, write factor {wr_f:.3f}")
    print()
    print("\n".join(out2))
    if out3:
        print()
        print("Prefill step (OPT-13B W6A6), DRAM bytes per launch:")
        print()
        print("\n".join(out3))
    if out4:
        print()
        print("Prefill step (OPT-13B W6A6), what the K loop waits on (mean over the run's launches):")
        print()
        print("\n".join(out4))


def copy_probe(torch):
    """A plain device copy of exactly 1 GiB (read 1 GiB, write 1 GiB)."""
    n = 1 << 30
    a = torch.empty(n, dtype=torch.uint8, device="cuda")
    a.fill_(1)
    b = torch.empty_like(a)
    torch.cuda.synchronize()
    for _ in range(3):
        b.copy_(a)
    torch.cuda.synchronize()
    print(json.dumps({"copy_probe_bytes_read": n, "copy_probe_bytes_written": n, "launches": 3}))


# (label, rows, channels, kernel) of the helper probe's launches, three each
HELPER_PROBE = [("ot_quantize_act, qkv/out/fc1 input", 4096, 5120, "quantize_act_kernel"),
                ("ot_quantize_act, fc2 input", 4096, 20480, "quantize_act_kernel"),
                ("ot_ln_quantize_act, qkv/fc1 LayerNorm", 4096, 5120, "ln_quantize_kernel")]


def helper_probe(torch, ot, synth, wl):
    """The activation quantizer and the fused LayerNorm on the OPT-13B W6A6
    shapes, three launches each, with a 1 GiB buffer written between launches
    so that each reads its input from HBM rather than the last-level cache."""
    flush = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
    K1 = wl.layers[0].K
    gamma, beta = (torch.from_numpy(a).cuda() for a in synth.ln_params(wl, 0))
    for label, M, K, kern in HELPER_PROBE:
        X = torch.randn(M, K, device="cuda").half()
        z = torch.zeros(K, device="cuda")
        inv_s = torch.full((K,), 4.0, device="cuda")
        Xq = torch.empty((M, K), dtype=torch.int8, device="cuda")
        for _ in range(3):
            flush.fill_(0)
            if kern == "ln_quantize_kernel":
                assert K == K1
                ot.ot_ln_quantize_act(X, gamma, beta, 1e-5, wl.a_bits, z, inv_s, Xq)
            else:
                ot.ot_quantize_act(X, wl.a_bits, z, inv_s, Xq)
        torch.cuda.synchronize()
    print(json.dumps({"helper_probe": [[lab, M, K] for lab, M, K, _ in HELPER_PROBE],
                      "launches_each": 3}))


def helper_traffic(d):
    """Markdown table of the helper probe's HBM-side bytes per launch, from
    FETCH_SIZE and WRITE_SIZE runs over `bench.py --helper-probe` (under
    d/helper_fetch, d/helper_write) scaled by the same counters on the 1 GiB
    copy (d/copy_fetch, d/copy_write).  Host only."""
    n_copy = 1 << 30
    factors = {}
    for c, sub in (("FETCH_SIZE", "copy_fetch"), ("WRITE_SIZE", "copy_write")):
        disp = _per_dispatch(_counter_rows(os.path.join(d, sub), c), "copyBuffer")
        kib = [v for _, v in disp if v > 0.5 * n_copy / 1024 / 4]
        factors[c] = n_copy / 1024 / float(np.median(kib))
    got, ns = {}, {}
    for c, sub in (("FETCH_SIZE", "helper_fetch"), ("WRITE_SIZE", "helper_write")):
        rows = _counter_rows(os.path.join(d, sub), c)
        q = [v for _, v in _per_dispatch(rows, "quantize_act_kernel")]
        ln = [v for _, v in _per_dispatch(rows, "ln_quantize_kernel")]
        if len(q) != 6 or len(ln) != 3:
            raise SystemExit(f"{sub}: {len(q)} quantizer and {len(ln)} LayerNorm dispatches, "
                             "expected 6 and 3")
        got[c] = [q[:3], q[3:], ln]
        for r in rows:  # each dispatch's own duration, both runs
            if "quantize_act_kernel" in r["Kernel_Name"] or "ln_quantize_kernel" in r["Kernel_Name"]:
                ns[(sub, int(r["Dispatch_Id"]))] = (r["Kernel_Name"],
                                                    int(r["End_Timestamp"]) - int(r["Start_Timestamp"]))
    dur = [[], [], []]
    for sub in ("helper_fetch", "helper_write"):
        ds = [v for k, v in sorted(ns.items()) if k[0] == sub]
        qs = [t for n, t in ds if "quantize_act_kernel" in n]
        dur[0] += qs[:3]
        dur[1] += qs[3:]
        dur[2] += [t for n, t in ds if "ln_quantize_kernel" in n]
    out = [f"Calibration on the 1 GiB copy: FETCH_SIZE factor {factors['FETCH_SIZE']:.3f}, "
           f"WRITE_SIZE factor {factors['WRITE_SIZE']:.3f} (bytes = KiB x 1024 x factor).", "",
           "| Launch | rows x channels | read bytes | written bytes | algorithmic read / written | "
           "read / algorithmic | written / algorithmic | us per launch (median of 6, under the "
           "profiler) | algorithmic GB/s |",
           "|---|---|---|---|---|---|---|---|---|"]
    for i, (label, M, K, kern) in enumerate(HELPER_PROBE):
        rd = float(np.mean(got["FETCH_SIZE"][i])) * 1024 * factors["FETCH_SIZE"]
        wr = float(np.mean(got["WRITE_SIZE"][i])) * 1024 * factors["WRITE_SIZE"]
        params = 12 * K if kern == "ln_quantize_kernel" else 8 * K  # gamma, beta, z, 1/s
        a_rd, a_wr = 2 * M * K + params, M * K
        us = float(np.median(dur[i])) / 1e3
        out.append(f"| {label} | {M} x {K} | {rd / 1e6:.1f} MB | {wr / 1e6:.1f} MB | "
                   f"{a_rd / 1e6:.1f} / {a_wr / 1e6:.1f} MB | {rd / a_rd:.3f} | {wr / a_wr:.3f} | "
                   f"{us:.1f} | {(a_rd + a_wr) / (us * 1e-6) / 1e9:.0f} |")
    print("\n".join(out))


def hbm_copy_context(torch, iters=10):
    """A plain 1 GiB device-to-device copy (torch's), for context: bytes read
    plus written per second."""
    n = 1 << 30
    a = torch.empty(n, dtype=torch.uint8, device="cuda")
    a.fill_(1)
    b = torch.empty_like(a)
    med, _, _ = median_ms(torch, lambda: b.copy_(a), iters)
    del a, b
    return dict(bytes_read_and_written=2 * n, ms=med, GBps=2 * n / (med * 1e-3) / 1e9)


def cpu_baseline(ot_oracle, layers, M, budget_s=10.0):
    """The oracle's quantize + integer GEMM + epilogue on the first R token
    rows of every linear, R doubled until the sample takes `budget_s`."""
    host = [dict(X=L["X"].cpu().numpy(), z=L["z"].cpu().numpy(), inv_s=L["inv_s"].cpu().numpy(),
                 Wq=L["Wq"].cpu().numpy(), sW=L["sW"].cpu().numpy(), bp=L["bp"].cpu().numpy(),
                 K=L["K"], N=L["N"]) for L in layers]
    a_bits = layers[0]["a_bits"]
    R = 64
    while True:
        t0 = time.perf_counter()
        for h in host:
            xq = ot_oracle.quantize_act(h["X"][:R], h["z"], h["inv_s"], a_bits)
            ot_oracle.epilogue(ot_oracle.int_gemm(xq, h["Wq"]), h["sW"], h["bp"])
        dt = time.perf_counter() - t0
        if dt >= budget_s or R >= M:
            break
        R = min(M, R * 2)
    ops = sum(2.0 * R * h["N"] * h["K"] for h in host)
    threads = None
    try:
        import threadpoolctl
        threads = max(i.get("num_threads", 0) for i in threadpoolctl.threadpool_info()) or None
    except Exception:
        pass
    return dict(value=ops / dt / 1e12, unit="TOPS", cores=threads or os.cpu_count(),
                kind="oracle", seconds=dt,
                sample=f"first {R} of {M} token rows of each of the 4 linears: quantize_act + "
                       f"int_gemm (fp64 BLAS) + epilogue; host os.cpu_count()={os.cpu_count()}")


# ---------------------------------------------------------------------------
def shader_clock_window(torch, step, seconds=1.0):
    """The shader clock while the prefill step runs back to back for about
    `seconds` (outside the timed region): the per-XCD current gfx clocks of
    the SMU's metrics table, read in-process through the amdsmi library
    every 5 ms by a thread (no subprocess), idle readings (< 500 MHz)
    dropped.  Returns an "error" entry instead where the library is
    missing or refuses."""
    import threading
    try:
        import amdsmi
        amdsmi.amdsmi_init(amdsmi.AmdSmiInitFlags.INIT_AMD_GPUS)
    except Exception as e:  # no SMI library or no access: report, do not fail
        return {"error": f"amdsmi unavailable: {e}"}
    try:
        h = amdsmi.amdsmi_get_processor_handles()[0]
        samples, stop = [], threading.Event()

        def sample():
            while not stop.is_set():
                clks = amdsmi.amdsmi_get_gpu_metrics_info(h).get("current_gfxclks")
                if isinstance(clks, list):
                    samples.append([c for c in clks if isinstance(c, int) and c >= 500])
                stop.wait(0.005)

        th = threading.Thread(target=sample, daemon=True)
        th.start()
        t0, runs = time.perf_counter(), 0
        while time.perf_counter() - t0 < seconds:
            for _ in range(10):
                step()
            torch.cuda.synchronize()
            runs += 10
        stop.set()
        th.join()
        flat = [c for row in samples for c in row]
        if not flat:
            return {"error": "no clock readings above idle"}
        per_xcd = [float(np.median([row[i] for row in samples if len(row) > i]))
                   for i in range(max(len(r) for r in samples))]
        return {"median_MHz": float(np.median(flat)), "p10_MHz": float(np.percentile(flat, 10)),
                "p90_MHz": float(np.percentile(flat, 90)), "per_xcd_median_MHz": per_xcd,
                "readings": len(samples), "steps": runs,
                "source": "amdsmi gpu metrics current_gfxclks, every 5 ms over back-to-back steps"}
    except Exception as e:
        return {"error": f"amdsmi read failed: {e}"}
    finally:
        try:
            amdsmi.amdsmi_shut_down()
        except Exception:
            pass


def time_prefill_step(torch, ot, wl, layers, steps, warmup):
    """The timed prefill step: for each linear, ot_quantize_act then
    ot_qlinear, `warmup` untimed steps, then `steps` steps between two events
    (ms per step), with an event pair around every ot_qlinear (mean ms per
    linear).  Returns (step function, ms per step, per-linear ms, wall s)."""
    nl = len(layers)
    ev_q = [[(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
             for _ in range(nl)] for _ in range(steps)]

    def step(events=None):
        for i, L in enumerate(layers):
            ot.ot_quantize_act(L["X"], wl.a_bits, L["z"], L["inv_s"], L["Xq"])
            if events is not None:
                events[i][0].record()
            ot.ot_qlinear(L["Xq"], L["Wq"], L["sW"], L["bp"], wl.a_bits, wl.w_bits, L["Y"])
            if events is not None:
                events[i][1].record()

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    t0 = time.perf_counter()
    start.record()
    for k in range(steps):
        step(ev_q[k])
    end.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms_step = start.elapsed_time(end) / steps
    per_layer_ms = [float(np.mean([ev_q[k][i][0].elapsed_time(ev_q[k][i][1])
                                   for k in range(steps)])) for i in range(nl)]
    return step, ms_step, per_layer_ms, wall


def with_buffers(torch, wl, layers, M):
    for L in layers:
        L["a_bits"] = wl.a_bits
        L["Xq"] = torch.empty((M, L["K"]), dtype=torch.int8, device="cuda")
        L["Y"] = torch.empty((M, L["N"]), dtype=torch.float16, device="cuda")
    return layers


# The paper's own speed and memory figures (Sec. 4.3, Fig. 3 and Table 5),
# measured end to end on whole OPT models on the hardware it names (two
# NVIDIA A100 GPUs, the variant not stated), against FP16: context for the
# per-linear figures here, not a target.
PAPER_CONTEXT = {
    "hardware": "2x NVIDIA A100 (as the paper states it), PyTorch",
    "end_to_end_speedup_vs_fp16": {"opt6.7b": 1.38, "opt13b": 1.48,
                                   "workload": "batch 1, 512 tokens (Sec. 4.3, Fig. 3)"},
    "memory_vs_fp16": "about 2x smaller (Sec. 4.3)",
    "decode_ms_per_token_fp16_to_ours": {"opt6.7b_bs8": [12.1, 8.2], "opt6.7b_bs16": [11.2, 8.1],
                                         "opt13b_bs8": [21.9, 15.6], "opt13b_bs16": [19.1, 14.3],
                                         "workload": "128-token sequences (Table 5)"},
}


def other_prefill_report(torch, ot, synth, name, pool, steps, warmup, iters, with_fp16):
    """Another prefill workload's four-linear step, timed like the headline
    one: GEMM TOPS and fraction of the int8 peak per linear and in total,
    the step with quantization, torch's fp16 linear on the same shapes
    (speedup) and the weight memory against fp16 (int8 codes + fp32 sW and
    b' against fp16 W and b)."""
    wl = synth.WORKLOADS[name]
    M = wl.M
    t0 = time.perf_counter()
    layers = with_buffers(torch, wl, prepare(wl, M, torch, ot, synth, pool), M)
    log(f"setup {name} {time.perf_counter() - t0:.1f}s")
    _, ms_step, per_layer_ms, _ = time_prefill_step(torch, ot, wl, layers, steps, warmup)
    ops = {L["name"]: 2.0 * M * L["N"] * L["K"] for L in layers}
    gemm_ms = sum(per_layer_ms)
    gemm_tops = sum(ops.values()) / (gemm_ms * 1e-3) / 1e12
    rec = {
        "tokens": M, "a_bits": wl.a_bits, "w_bits": wl.w_bits,
        "layers": {L["name"]: [L["K"], L["N"]] for L in layers},
        "plan": {L["name"]: ot.ot_qlinear_plan(M, L["N"], L["K"]) for L in layers},
        "qlinear_ms_per_launch": {L["name"]: round(t, 4) for L, t in zip(layers, per_layer_ms)},
        "qlinear_frac_of_int8_peak_per_launch": {
            L["name"]: round(ops[L["name"]] / (t * 1e-3) / 1e12 / PEAK_INT8_TOPS, 4)
            for L, t in zip(layers, per_layer_ms)},
        "qlinear_ms": round(gemm_ms, 4),
        "qlinear_tops": round(gemm_tops, 1),
        "qlinear_frac_of_int8_peak": round(gemm_tops / PEAK_INT8_TOPS, 4),
        "step_ms": round(ms_step, 4),
        "step_tops": round(sum(ops.values()) / (ms_step * 1e-3) / 1e12, 1),
        "tokens_per_s": round(M / (ms_step * 1e-3), 1),
        "weight_bytes": sum(L["K"] * L["N"] + 8 * L["N"] for L in layers),
        "fp16_weight_bytes": sum(2 * L["K"] * L["N"] + 2 * L["N"] for L in layers),
    }
    rec["weight_memory_ratio_vs_fp16"] = round(rec["fp16_weight_bytes"] / rec["weight_bytes"], 4)
    if with_fp16:
        fb = fp16_baseline(torch, layers, M, iters)
        rec["fp16_linear_ms"] = round(fb["ms_per_stack"], 4)
        rec["fp16_linear_tflops"] = round(fb["tflops"], 1)
        rec["speedup_of_step_vs_fp16"] = round(fb["ms_per_stack"] / ms_step, 4)
        rec["speedup_of_qlinear_vs_fp16"] = round(fb["ms_per_stack"] / gemm_ms, 4)
    log(f"{name}: qlinear {gemm_ms:.3f} ms ({gemm_tops:.0f} TOPS, "
        f"{100 * gemm_tops / PEAK_INT8_TOPS:.1f} % of peak); step {ms_step:.3f} ms"
        + (f"; fp16 {rec['fp16_linear_ms']:.3f} ms" if with_fp16 else ""))
    layers.clear()
    torch.cuda.empty_cache()
    return rec


def main():
    args = parse()
    if args.traffic_record:
        traffic_record(args.traffic_record, args.workload)
        return
    if args.counter_summary:
        counter_summary(args.counter_summary, args.workload, args.decode_workload)
        return
    if args.helper_traffic:
        helper_traffic(args.helper_traffic)
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (got --gpus {args.gpus}); the quantized linear "
              "is single-device here and no multi-GPU path is built.", file=sys.stderr)
        sys.exit(2)
    import torch

    from paper_2406_18832_amd import ot, synth
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    if args.copy_probe:
        copy_probe(torch)
        return
    if args.helper_probe:
        helper_probe(torch, ot, synth, synth.WORKLOADS[args.workload])
        return
    if args.decode_probe:
        ot.lib()
        pool = cf.ThreadPoolExecutor(max_workers=min(16, os.cpu_count() or 4))
        decode_probe(torch, ot, synth, synth.WORKLOADS[args.decode_workload], pool)
        pool.shutdown()
        return
    if args.quality:
        from paper_2406_18832_amd import quality
        ot.lib()
        recs = quality.sweep(log=log)
        print(json.dumps({"quality_sweep": recs}), flush=True)
        return
    ot.lib()
    wl = synth.WORKLOADS[args.workload]
    M = wl.M
    pool = cf.ThreadPoolExecutor(max_workers=min(16, os.cpu_count() or 4))
    t_setup = time.perf_counter()
    layers = with_buffers(torch, wl, prepare(wl, M, torch, ot, synth, pool), M)
    log(f"setup {time.perf_counter() - t_setup:.1f}s")

    step, ms_step, per_layer_ms, wall = time_prefill_step(torch, ot, wl, layers, args.steps,
                                                          args.warmup)
    ops_step = sum(2.0 * M * L["N"] * L["K"] for L in layers)
    tops = ops_step / (ms_step * 1e-3) / 1e12
    gemm_ms = sum(per_layer_ms)
    gemm_tops = ops_step / (gemm_ms * 1e-3) / 1e12
    log(f"step {ms_step:.3f} ms ({tops:.0f} TOPS); qlinear {gemm_ms:.3f} ms ({gemm_tops:.0f} TOPS); "
        f"wall {wall:.2f}s")

    result = {
        "metric": METRIC,
        "value": round(tops, 2),
        "unit": "TOPS",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "int8",
        "data": "synthetic",
        "config": {"workload": wl.name, "tokens": M, "a_bits": wl.a_bits, "w_bits": wl.w_bits,
                   "layers": {L["name"]: [L["K"], L["N"]] for L in layers},
                   "step": "4 x (ot_quantize_act + ot_qlinear)"},
        "roofline": {"bound": "mfma", "kernel": "qgemm_prefill",
                     "achieved": round(gemm_tops, 2), "peak": PEAK_INT8_TOPS, "unit": "TOP/s",
                     "frac": round(gemm_tops / PEAK_INT8_TOPS, 4), "traffic": measured_traffic(),
                     "ops_per_launch": {L["name"]: 2 * M * L["N"] * L["K"] for L in layers},
                     "ms_per_launch": {L["name"]: round(t, 4) for L, t in zip(layers, per_layer_ms)}},
        "qlinear_tops": round(gemm_tops, 2),
        "quantize_act_ms_per_step": round(ms_step - gemm_ms, 4),
        "tokens_per_s": round(M / (ms_step * 1e-3), 1),
    }
    if not args.no_sclk:
        clk = shader_clock_window(torch, step)
        if "median_MHz" in clk:
            clk["frac_of_2400_MHz"] = round(clk["median_MHz"] / 2400.0, 4)
            # What the SMU reports is not the clock the GEMM's waves run at:
            # counted inside the kernels (shader cycles over the 100 MHz
            # real-time counter, and GRBM_GUI_ACTIVE over each dispatch's
            # duration) the prefill GEMMs run at 1.7-2.1 GHz.
            clk["note"] = ("SMU-reported clock; the GEMM dispatches' own cycle counts give "
                           "1.7-2.1 GHz (counter summary under profiles/)")
            log(f"SMU-reported shader clock over {clk['steps']} steps: median "
                f"{clk['median_MHz']:.0f} MHz")
        else:
            log(f"shader clock: {clk['error']}")
        result["prefill_smu_clock"] = clk
    if not args.no_fp16:
        fb = fp16_baseline(torch, layers, M, args.iters)
        fb["speedup_of_step"] = fb["ms_per_stack"] / ms_step
        fb["weight_bytes_ratio"] = (sum(2 * L["K"] * L["N"] + 2 * L["N"] for L in layers) /
                                    sum(L["K"] * L["N"] + 8 * L["N"] for L in layers))
        result["fp16_baseline"] = fb
        log(f"fp16 linear stack {fb['ms_per_stack']:.3f} ms ({fb['tflops']:.0f} TFLOPs)")
    if not args.no_mixed:
        result["mixed_block"] = mixed_block_report(torch, ot, wl, layers, args.iters)
    if not args.no_asym:
        result["asym_weights"] = asym_report(torch, ot, wl, layers, args.iters)
    if not args.no_cpu:
        from oracle import ot_oracle
        result["cpu_baseline"] = cpu_baseline(ot_oracle, layers, M)
        log(f"cpu oracle {result['cpu_baseline']['value']:.3f} TOPS")
    for L in layers:
        del L["W16"]
    if not args.no_ln:
        result["ln_quantize"] = {"workload": wl.name, "bound": "hbm", "peak_GBps": PEAK_HBM_GBS,
                                 "kernel": "ln_quantize_kernel",
                                 "by_layer": ln_quantize_report(torch, ot, synth, wl, args.iters)}
    layers.clear()
    torch.cuda.empty_cache()
    if not args.no_other:
        result["other_prefill"] = {
            n: other_prefill_report(torch, ot, synth, n, pool, args.steps, args.warmup,
                                    args.iters, not args.no_fp16)
            for n in ("opt6.7b_w8a8", "opt66b_w8a8") if n != wl.name}
        result["paper_context"] = PAPER_CONTEXT
    if not args.no_decode:
        dwl = synth.WORKLOADS[args.decode_workload]
        result["decode"] = {"workload": dwl.name, "bound": "hbm", "peak_GBps": PEAK_HBM_GBS,
                            "by_M": decode_report(torch, ot, synth, dwl, pool, args.iters,
                                                  not args.no_fp16)}
        # per token count, the faster of the two weight layouts (eager launches)
        summ = {}
        for m, r in result["decode"]["by_M"].items():
            packed = r.get("packed_us_per_stack")
            best = "packed" if packed is not None and packed < r["us_per_stack"] else "row-major"
            us = packed if best == "packed" else r["us_per_stack"]
            gbs = r["bytes_per_stack"] / (us * 1e-6) / 1e9
            summ[m] = {"weights": best, "us_per_stack": round(us, 2), "GBps": round(gbs, 1),
                       "frac_of_hbm_peak": round(gbs / PEAK_HBM_GBS, 4)}
        result["decode"]["best_layout_by_M"] = summ
        torch.cuda.empty_cache()
        result["decode"]["hbm_copy_context"] = hbm_copy_context(torch)
        log(f"plain 1 GiB device copy: {result['decode']['hbm_copy_context']['GBps']:.0f} GB/s "
            f"(read + write)")
    pool.shutdown()
    # provenance: the loaded library's own record of its sources, checked
    # against the tree this run came from
    result["library"] = ot.build_info()
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
