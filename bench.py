"""Benchmark: Gated DeltaNet prefill + decode on one MI355X.

One step = one gdn_prefill over the 4096-token workload (1 sequence, 16 q/k
heads, 32 v heads, d = 128, chunk 64, bf16) plus one gdn_decode over the
batch-64 workload (same heads, fp32 state updated in place). Inputs are
resident in HBM before the timed region; three input sets are rotated so
that consecutive calls never re-read data the 256 MB Infinity Cache could
still hold. The prefill calls share one workspace, as a caller that sizes it
once for its largest batch would (with a fresh workspace per input set the
call is about 10% slower: the per-chunk tables then land on cold lines). The K prefill calls and the K decode calls each run back to back
between HIP events on the stream they are launched on.

Prints one JSON line. `value` is prefill tokens/s (sum of the timed prefill
calls); decode latency and HBM rate ride alongside. Roofline figures use
fixed algorithmic counts:
  prefill flop per token per value head = 6 d^2 + (6 + 4 HQK/HV) C d + C^2/3
  prefill bytes = T (2 HQK d e + 2 HV d e + 8 HV) + N HV d^2 4 (1 + [S0])
                  + 4 (N + 1)
  decode bytes  = 2 B HV d^2 4 + B (2 HQK + 2 HV) d 2 + 8 B HV
`traffic` is the counter-measured byte count per launch (see MEASURED_TRAFFIC).

Alongside: the per-call spread (`us_per_call_dist`, `us_per_step_dist`: p10,
p50, p90 over 100 calls, each between its own events), `decode_latency_us`
(one decode step per batch size, graph-replayed), `prefill_dispatch`
(short-sequence batches: the library's chunk choice against the fixed 64-token
chunk) and `prefill_other_workloads` (the 66K-token varlen batch and the
2 x 32768-token prefill).
"""
import argparse
import glob
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0          # MI355X HBM3E
PEAK_BF16_TFLOPS = 2500.0      # MI355X dense bf16 matrix peak
METRIC = "prefill tokens/sec + MFMA util; decode µs/step + achieved HBM GB/s"


# Bytes moved per launch as the memory counters read them (FETCH_SIZE and
# WRITE_SIZE passes, each scaled by what the counter reads for a copy of known
# size; profiles/prefill4k_decode64_memory_counters.md), keyed by a hash of
# the kernel sources they were taken on. Any change to those sources makes
# the figures stale, and `traffic` is then reported as null.
MEASURED_TRAFFIC = {
    "123ea7c4416aacf9c32a092558d420547017f93859093c0be34197462721dbe7":
        {"prefill": 219674852, "decode": 274395845},
}


def kernel_source_hash():
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2607_16831_amd", "csrc")
    for f in sorted(glob.glob(os.path.join(csrc, "*.hip")) + glob.glob(os.path.join(csrc, "*.h"))):
        h.update(os.path.basename(f).encode())
        with open(f, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def prefill_flops(T, hqk, hv, d, C):
    return float(T) * hv * (6 * d * d + (6 + 4.0 * hqk / hv) * C * d + C * C / 3.0)


def prefill_flops_executed(T, hqk, hv, d, C):
    """Products the kernels run in the R form (U = T'(V - exp(gamma) K S^T),
    no W = T'(beta Gamma K)): 6 d^2 (K S^T, Q S^T, the state update) +
    4 C d (T' Y and P U) + 4 (HQK/HV) C d (the two Gram products, shared by
    a key head's value heads) + C^2/3 (the triangular factor) per token and
    value head. The fixed formula above also counts the W product (2 C d)."""
    return float(T) * hv * (6 * d * d + (4 + 4.0 * hqk / hv) * C * d + C * C / 3.0)


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    import platform
    return platform.processor() or platform.machine()


def prefill_bytes(T, N, hqk, hv, d, e, has_s0):
    return (T * (2 * hqk * d * e + 2 * hv * d * e + 8 * hv)
            + N * hv * d * d * 4 * (1 + int(has_s0)) + 4 * (N + 1))


def decode_bytes(B, hqk, hv, d):
    return 2 * B * hv * d * d * 4 + B * (2 * hqk + 2 * hv) * d * 2 + 8 * B * hv


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=30)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--rotate", type=int, default=3)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=10.0)
    ap.add_argument("--no-decode-sweep", action="store_true",
                    help="skip the small-batch decode latency sweep")
    ap.add_argument("--no-other-workloads", action="store_true",
                    help="skip timing the 66K-token varlen batch and the 2 x 32768-token prefill")
    ap.add_argument("--no-dispatch-sweep", action="store_true",
                    help="skip the prefill shape-dispatch comparison over short-sequence batches")
    ap.add_argument("--segment", type=int, default=0, metavar="L",
                    help="force segments of L chunks in the prefill's whole-chain carry "
                         "(0: the library's choice)")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MB",
                    help="before warm-up, run a read-once/write-once kernel over MB "
                         "megabytes (three times), whose memory counters calibrate "
                         "FETCH_SIZE / WRITE_SIZE")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py: this build runs on one GPU only (the recurrence has no "
              "cross-GPU step here); use --gpus 1", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2607_16831_amd import gdn, synth

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    dev = torch.device("cuda:0")
    wp, wd = synth.PREFILL_4K, synth.DECODE_B64
    pchunk = wp.chunk | (gdn.CHUNK_SEGMENT(args.segment) if args.segment > 0 else 0)

    # ---------------------------------------------------------------- inputs
    P, D = [], []
    for r in range(args.rotate):
        x = synth.make(wp, seed=wp.seed + 100 * r)
        s = {k: (v.to(dev) if isinstance(v, torch.Tensor) else v) for k, v in x.items()}
        T = s["q"].shape[0]
        s["o"] = torch.empty((T, wp.hv, wp.d), dtype=torch.bfloat16, device=dev)
        s["fs"] = torch.empty((wp.n_seqs, wp.hv, wp.d, wp.d), device=dev)
        s["ws"] = P[0]["ws"] if P else gdn.alloc_workspace(wp.n_seqs, T, wp.hqk, wp.hv, wp.d,
                                                             pchunk, dev)
        P.append(s)
        y = synth.make(wd, seed=wd.seed + 100 * r)
        t = {k: (v.to(dev) if isinstance(v, torch.Tensor) else v) for k, v in y.items()}
        t["o"] = torch.empty((wd.n_seqs, wd.hv, wd.d), dtype=torch.bfloat16, device=dev)
        D.append(t)
    torch.cuda.synchronize()

    if args.copy_calibration > 0:
        n = args.copy_calibration * (1 << 20) // 4
        src = torch.ones(n, device=dev)
        dst = torch.empty_like(src)
        for _ in range(3):
            torch.neg(src, out=dst)  # reads n*4 bytes, writes n*4 bytes
        torch.cuda.synchronize()
        del src, dst

    def run_prefill(s):
        gdn.prefill(s["q"], s["k"], s["v"], s["g"], s["beta"], s["cu_seqlens"],
                    initial_state=s["initial_state"], chunk=pchunk, o=s["o"],
                    final_state=s["fs"], workspace=s["ws"])

    def run_decode(t):
        gdn.decode(t["q"], t["k"], t["v"], t["g"], t["beta"], t["initial_state"], o=t["o"])

    for i in range(args.warmup):
        run_prefill(P[i % args.rotate])
        run_decode(D[i % args.rotate])
    torch.cuda.synchronize()

    # ---------------------------------------------------------------- timed
    # K steps: the K prefill calls back to back, then the K decode calls back
    # to back, each batch bracketed by events on the launch stream, so the
    # per-call averages carry no per-call event overhead.
    K = args.steps
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    ev[0].record()
    for i in range(K):
        run_prefill(P[i % args.rotate])
    ev[1].record()
    for i in range(K):
        run_decode(D[i % args.rotate])
    ev[2].record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_start

    # The same K prefill calls with a workspace per input set: the per-chunk
    # tables then never land on lines the previous call left in the caches.
    wss = [P[0]["ws"]] + [torch.empty_like(P[0]["ws"]) for _ in range(1, args.rotate)]
    for i in range(args.rotate):
        run_prefill(dict(P[i], ws=wss[i]))
    torch.cuda.synchronize()
    ec = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    ec[0].record()
    for i in range(K):
        run_prefill(dict(P[i % args.rotate], ws=wss[i % args.rotate]))
    ec[1].record()
    torch.cuda.synchronize()
    pre_cold_avg = ec[0].elapsed_time(ec[1]) / 1e3 / K
    del wss

    # Per-call spread: 100 prefill calls, then 100 decode steps, each between
    # a pair of events of its own (rotating input sets, shared workspace).
    def per_call(fn, items, n=100):
        evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
               for _ in range(n)]
        for i in range(n):
            evs[i][0].record()
            fn(items[i % len(items)])
            evs[i][1].record()
        torch.cuda.synchronize()
        ts = sorted(a.elapsed_time(b) * 1e3 for a, b in evs)
        return {"calls": n, "p10": round(ts[n // 10], 2), "p50": round(ts[n // 2], 2),
                "p90": round(ts[(9 * n) // 10], 2)}
    pre_dist = per_call(run_prefill, P)
    dec_dist = per_call(run_decode, D)

    pre_s = ev[0].elapsed_time(ev[1]) / 1e3
    dec_s = ev[1].elapsed_time(ev[2]) / 1e3
    T = P[0]["q"].shape[0]
    pre_avg = pre_s / K
    dec_avg = dec_s / K
    pre_tps = K * T / pre_s
    flop = prefill_flops(T, wp.hqk, wp.hv, wp.d, wp.chunk)
    flop_exec = prefill_flops_executed(T, wp.hqk, wp.hv, wp.d, wp.chunk)
    pbytes = prefill_bytes(T, wp.n_seqs, wp.hqk, wp.hv, wp.d, 2, False)
    dbytes = decode_bytes(wd.n_seqs, wd.hqk, wd.hv, wd.d)
    pre_tflops = flop / pre_avg / 1e12
    dec_gbs = dbytes / dec_avg / 1e9

    measured = MEASURED_TRAFFIC.get(kernel_source_hash())
    roof_pre = {"bound": "mfma", "achieved": round(pre_tflops, 2),
                "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                "frac": round(pre_tflops / PEAK_BF16_TFLOPS, 4),
                "traffic": measured["prefill"] if measured else None,
                "kernel": "gdn_prefill (chunk_local + chunk_carry)",
                "algorithmic_flop_per_launch": flop,
                "executed_flop_per_launch": flop_exec,
                "frac_executed": round(flop_exec / pre_avg / 1e12 / PEAK_BF16_TFLOPS, 4),
                "hbm_view_gbs": round(pbytes / pre_avg / 1e9, 1)}
    roof_dec = {"bound": "hbm", "achieved": round(dec_gbs, 1), "peak": PEAK_HBM_GBS,
                "unit": "GB/s", "frac": round(dec_gbs / PEAK_HBM_GBS, 4),
                "traffic": measured["decode"] if measured else None,
                "kernel": "decode_kernel<128, bf16>",
                "algorithmic_bytes_per_launch": dbytes}
    dominant = roof_dec if dec_avg >= pre_avg else roof_pre

    out = {
        "metric": METRIC, "value": round(pre_tps, 1), "unit": "tokens/s",
        "n_gpus": 1, "steps": K, "warmup": args.warmup,
        "ms_per_step": round(wall * 1e3 / K, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": "prefill %s + decode %s" % (wp.name, wd.name),
                   "prefill_tokens": T, "decode_batch": wd.n_seqs,
                   "heads_qk_v": [wp.hqk, wp.hv], "d": wp.d, "chunk": wp.chunk,
                   "rotating_input_sets": args.rotate},
        "prefill": {"us_per_call": round(pre_avg * 1e6, 2),
                    "us_per_call_workspace_per_set": round(pre_cold_avg * 1e6, 2),
                    "tokens_per_s": round(pre_tps, 1), "tflops": round(pre_tflops, 2),
                    "mfma_util": round(pre_tflops / PEAK_BF16_TFLOPS, 4),
                    "us_per_call_dist": pre_dist},
        "decode": {"us_per_step": round(dec_avg * 1e6, 2),
                   "hbm_gbs": round(dec_gbs, 1), "hbm_frac": round(dec_gbs / PEAK_HBM_GBS, 4),
                   "us_per_step_dist": dec_dist},
        "roofline": dominant,
        "rooflines": [roof_pre, roof_dec],
    }

    # ---------------------------------------------------- small-batch decode
    # Latency of one decode step per batch size (same heads and d), from cold
    # state: each step advances a different state buffer, rotating over
    # enough buffers (at least 3, and at least 3 x 256 MiB in all) that the
    # Infinity Cache cannot hold the state between its visits. The steps are
    # captured in a HIP graph and replayed, so the time per step is the
    # kernel's, without the host launch path of the Python binding. The warm
    # figure (one state buffer, 20 steps) rides alongside.
    if not args.no_decode_sweep:
        lat, warm, cold_frac = {}, {}, {}
        for B in (1, 8, 16, 48, 64):
            w = wd.replace(n_seqs=B, seed=wd.seed + 7)
            y = synth.make(w)
            t = {k: (v.to(dev) if isinstance(v, torch.Tensor) else v) for k, v in y.items()}
            t["o"] = torch.empty((B, w.hv, w.d), dtype=torch.bfloat16, device=dev)
            sbytes = t["initial_state"].numel() * 4
            nset = max(3, -(-3 * (256 << 20) // sbytes))
            states = [t["initial_state"].clone() for _ in range(nset)]

            def graph_time(sts, reps):
                for st in sts[:3]:
                    run_decode(dict(t, initial_state=st))
                torch.cuda.synchronize()
                graph = torch.cuda.CUDAGraph()
                with torch.cuda.graph(graph):
                    for st in sts:
                        run_decode(dict(t, initial_state=st))
                graph.replay()
                torch.cuda.synchronize()
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record()
                for _ in range(reps):
                    graph.replay()
                e1.record()
                torch.cuda.synchronize()
                del graph
                return e0.elapsed_time(e1) * 1e3 / (reps * len(sts))

            lat[str(B)] = round(graph_time(states, 3), 2)
            warm[str(B)] = round(graph_time([t["initial_state"]] * 20, 5), 2)
            cold_frac[str(B)] = round(decode_bytes(B, w.hqk, w.hv, w.d) / (lat[str(B)] * 1e-6)
                                      / 1e9 / PEAK_HBM_GBS, 4)
            del states, t
        out["decode_latency_us"] = lat
        out["decode_latency_hbm_frac"] = cold_frac
        out["decode_latency_warm_us"] = warm

    # ------------------------------------------------- prefill shape dispatch
    # Batches of N equal-length sequences (same heads, d and dtype as the
    # main workload, no initial state): time per call with the library's own
    # choice (chunk = 0) against the fixed 64-token chunk, 20 calls between
    # events after 3 warm-up calls, one input set per shape.
    if not args.no_dispatch_sweep:
        disp = {}
        for N, L in ((1024, 1), (512, 4), (256, 8), (128, 16), (64, 32), (16, 256),
                     (2, 2048)):
            w = wp.replace(seq_len=L, n_seqs=N, seed=wp.seed + 11)
            y = synth.make(w)
            t = {k: (v.to(dev) if isinstance(v, torch.Tensor) else v) for k, v in y.items()}
            o = torch.empty((N * L, w.hv, w.d), dtype=torch.bfloat16, device=dev)
            fs = torch.empty((N, w.hv, w.d, w.d), device=dev)
            ws = gdn.alloc_workspace(N, N * L, w.hqk, w.hv, w.d, gdn.CHUNK_AUTO, dev)
            row = {"auto_chunk": gdn.prefill_auto_chunk(N, N * L, w.hqk, w.hv, w.d, w.d)}
            for key, c in (("auto", gdn.CHUNK_AUTO), ("chunk64", 64)):
                def call():
                    gdn.prefill(t["q"], t["k"], t["v"], t["g"], t["beta"], t["cu_seqlens"],
                                chunk=c, o=o, final_state=fs, workspace=ws)
                for _ in range(3):
                    call()
                torch.cuda.synchronize()
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record()
                for _ in range(20):
                    call()
                e1.record()
                torch.cuda.synchronize()
                row[key + "_us"] = round(e0.elapsed_time(e1) * 1e3 / 20, 2)
            row["auto_tokens_per_s"] = round(N * L / (row["auto_us"] * 1e-6), 1)
            disp["N%d_L%d" % (N, L)] = row
            del t, o, fs, ws
        out["prefill_dispatch"] = disp

    # ------------------------------------------------- larger prefill batches
    # The varlen batch (16 sequences, lengths U[64, 8192], nonzero initial
    # states) and the long-context pair (2 x 32768 tokens, strong decay), same
    # heads and d: time per call (events, 5 calls after 2 warm-up calls, one
    # input set each) with 64-token chunks, with the algorithmic flop count of
    # the same formula; then the same with the library's own chunk choice
    # (chunk = 0; the varlen batch fixes no chunk size) when it differs.
    if not args.no_other_workloads:
        other = {}
        for w in (synth.PREFILL_VARLEN, synth.PREFILL_LONG):
            y = synth.make(w)
            t = {k: (v.to(dev) if isinstance(v, torch.Tensor) else v) for k, v in y.items()}
            Tw = t["q"].shape[0]
            o = torch.empty((Tw, w.hv, w.d), dtype=torch.bfloat16, device=dev)
            fs = torch.empty((w.n_seqs, w.hv, w.d, w.d), device=dev)
            ws = gdn.alloc_workspace(w.n_seqs, Tw, w.hqk, w.hv, w.d, gdn.CHUNK_AUTO, dev)

            def time_chunk(chunk):
                def call():
                    gdn.prefill(t["q"], t["k"], t["v"], t["g"], t["beta"], t["cu_seqlens"],
                                initial_state=t["initial_state"], chunk=chunk, o=o,
                                final_state=fs, workspace=ws)
                for _ in range(2):
                    call()
                torch.cuda.synchronize()
                e0 = torch.cuda.Event(enable_timing=True)
                e1 = torch.cuda.Event(enable_timing=True)
                e0.record()
                for _ in range(5):
                    call()
                e1.record()
                torch.cuda.synchronize()
                return e0.elapsed_time(e1) * 1e3 / 5

            us = time_chunk(w.chunk)
            fl = prefill_flops(Tw, w.hqk, w.hv, w.d, w.chunk)
            row = {"tokens": Tw, "chunk": w.chunk, "us_per_call": round(us, 1),
                   "tokens_per_s": round(Tw / (us * 1e-6), 1),
                   "tflops": round(fl / (us * 1e-6) / 1e12, 2),
                   "mfma_util": round(fl / (us * 1e-6) / 1e12 / PEAK_BF16_TFLOPS, 4)}
            ca = gdn.prefill_auto_chunk(w.n_seqs, Tw, w.hqk, w.hv, w.d, w.d)
            row["auto_chunk"] = ca
            if ca != w.chunk:
                ua = time_chunk(gdn.CHUNK_AUTO)
                fa = prefill_flops(Tw, w.hqk, w.hv, w.d, ca)
                row.update({"us_per_call_auto": round(ua, 1),
                            "tokens_per_s_auto": round(Tw / (ua * 1e-6), 1),
                            "mfma_util_auto": round(fa / (ua * 1e-6) / 1e12 / PEAK_BF16_TFLOPS,
                                                    4)})
            other[w.name] = row
            del t, o, fs, ws
        out["prefill_other_workloads"] = other

    # ---------------------------------------------------------------- oracle
    if not args.no_cpu_baseline:
        import oracle
        x = synth.make(wp)
        reps, t0 = 0, time.perf_counter()
        while True:
            oracle.prefill(x["q"], x["k"], x["v"], x["g"], x["beta"], x["cu_seqlens"],
                           x["initial_state"])
            reps += 1
            el = time.perf_counter() - t0
            if el >= args.cpu_seconds:
                break
        out["cpu_baseline"] = {
            "value": round(reps * T / el, 1), "unit": "tokens/s",
            "cores": oracle.num_threads(), "kind": "oracle",
            "sample": "%d full runs of the 4096-token prefill (all 32 heads), fp64 "
                      "token-serial, %.1f s wall on %d threads of %s (%d logical CPUs)"
                      % (reps, el, oracle.num_threads(), cpu_model(), os.cpu_count() or 0),
            "cpu_model": cpu_model()}
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
