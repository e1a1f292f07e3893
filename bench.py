"""Benchmark of the capsule + chunked-scan hot path on one MI355X.

Workload (default): the 48-layer hybrid stack -- 36 gated linear-attention
layers (32 heads, dk = dv = 128) and 12 full-attention layers (4 KV heads,
d = 256, K and V bf16), prefix 16384, chunk 64, conv tails 4 x 4096 bf16 per
linear layer.  One step is one pass of the whole hot path:

  1. cold chunked prefill of the 36 linear layers, writing o and the state at
     every chunk boundary (the scan's full output)            -> scan tokens/s
  2. the same prefill writing only o and the final state (the cold-TTFT path)
  3. snapshot of the live set at P = 16384 (881,983,488 B)
  4. restore of that capsule into the live set                -> restore GB/s
  5. fork of the capsule into 4 sibling sessions (read once, write 4x)
  6. one continuation token through the 36 linear layers from the restored
     state (T = 1 prefill calls)

Every phase is bracketed by HIP events recorded on the stream the kernels run
on.  restore/cold TTFT = (phase 2 + phase 6) / (phase 4 + phase 6).

After the timed steps, outside them:
  * `ttft_ms`: 30 repeats of the cold leg (the 36 layers' chunked prefill
    with final states + the 12 full-attention layers' K/V rows materialised +
    the first token) and of the capsule leg (restore + the first token),
    p50 / p90 / p99;
  * `restore_decode_graph`: restore + first token as one HIP graph;
  * `host_tier`: demote / promote of the capsule over the host link;
  * `fp8_kv`: the K/V region in FP8 with bound bf16 working stages: restore
    into the same session (stage re-bound, nothing converted) and into
    another session (the first read converts all P rows);
  * `gdn`: one gated delta-rule layer of the same shape (the model family's
    Gated DeltaNet state);
  * `gather`: the robot episode reset (32 environments, a gallery of 8
    capsules, 1000 batched gather-restores);
  * `hybrid8`: the 8-layer workload -- its 14.8 MB capsule's restore
    latency, the 32 decode steps after a restore, cold vs capsule TTFT;
  * `cpu_baseline*`: the oracle on the host (see cpu_baseline).

The JSON line's `value` is the capsule restore bandwidth (GB/s, bytes read +
written); the scan and TTFT figures ride along as extra keys.  The scan's MFMA
figures: `scan_pct_mfma_useful` (useful flops / time / peak), its ceiling at
full HBM bandwidth, and `scan_pct_mfma_busy_counter`, the MFMA pipe's busy
fraction from rocprofv3 counters of the same kernel source.  `roofline`
covers the dominant kernel (the scan, phase 1); `roofline_copy`,
`roofline_snapshot` and `roofline_fork` the capsule copies, `gdn` and
`gather` carry their own.
Inputs are synthetic (synth module, fixed seeds); 4 distinct layers of q/k/v/g
are generated on the host and copied into the 36 layers' own device buffers.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0        # MI355X HBM3E, GB/s
MFMA_BF16_PEAK_TFS = 2500.0  # MI355X dense bf16 MFMA, TFLOP/s
LINK_PEAK_GBS = 64.0         # host link, PCIe 5.0 x16, one direction

# HBM bytes per launch from rocprofv3 FETCH_SIZE / WRITE_SIZE runs (FETCH_SIZE
# scaled by 1.99890 from the runtime's plain copies of known size); the
# counters belong to the kernel source with the given sha256 and are reported
# only while it is unchanged.  Summary and commands:
# profiles/hybrid48_hbm_traffic.md.
LINATTN_SRC = "paper_2606_20537_amd/csrc/linattn_scan.hip"
COPY_SRC = "paper_2606_20537_amd/csrc/capsule_copy.hip"
GDN_SRC = "paper_2606_20537_amd/csrc/gdn_scan.hip"
LINATTN_SHA = "09e420c2db0aea75d4aceb67e34dbe75c35c7f6ed39eb054bbbfd048226ade63"
COPY_SHA = "3fe58e0a55a7b15d596057bce3dc33d9409338b3d9d5d137fddb7f8da5978430"
GDN_SHA = "4cdea6657262021a85378f62e243eda289150d1bf653666fc2f29d5c485d6c54"
MEASURED_TRAFFIC = {
    "scan_cs": {"src": LINATTN_SRC, "sha256": LINATTN_SHA, "bytes": 1228826037},
    "restore": {"src": COPY_SRC, "sha256": COPY_SHA, "bytes": 1763625618},
    "snapshot": {"src": COPY_SRC, "sha256": COPY_SHA, "bytes": 1763688951},
    "fork4": {"src": COPY_SRC, "sha256": COPY_SHA, "bytes": 4409930338},
    "gather": {"src": COPY_SRC, "sha256": COPY_SHA, "bytes": 1010166192},
    "gdn": {"src": GDN_SRC, "sha256": GDN_SHA, "bytes": 1617845357},
}

# MFMA pipe busy from SQ_VALU_MFMA_BUSY_CYCLES / (1024 SIMDs x GRBM_GUI_ACTIVE
# / 8 XCDs), per scan launch on the 48-layer workload, with the same sha256
# guard.  Summary and commands: profiles/hybrid48_scan_counters.md.
MEASURED_MFMA_BUSY = {
    "scan_cs": {"src": LINATTN_SRC, "sha256": LINATTN_SHA, "frac": 0.1591},
    "scan_final": {"src": LINATTN_SRC, "sha256": LINATTN_SHA, "frac": 0.1918},
    "gdn_scan": {"src": GDN_SRC, "sha256": GDN_SHA, "frac": 0.1751},
}


def _src_unchanged(m):
    import hashlib
    with open(os.path.join(ROOT, m["src"]), "rb") as f:
        return hashlib.sha256(f.read()).hexdigest() == m["sha256"]


def measured_traffic(key):
    m = MEASURED_TRAFFIC[key]
    return m["bytes"] if _src_unchanged(m) else None


def measured_mfma_busy(key):
    m = MEASURED_MFMA_BUSY[key]
    return round(100 * m["frac"], 2) if _src_unchanged(m) else None


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="hybrid48")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--distinct-layers", type=int, default=4)
    return ap.parse_args()


def scan_bytes(T, H, dk, dv, chunk_states):
    """Algorithmic HBM bytes of one prefill launch (bf16 q,k,v; fp32 g, o,
    states; zero entering state)."""
    n_chunks = (T + 63) // 64
    b = T * H * (2 * (2 * dk + dv) + 4 + 4 * dv) + H * dk * dv * 4
    if chunk_states:
        b += n_chunks * H * dk * dv * 4
    return b


def gdn_bytes(T, H, dk, dv):
    """Algorithmic HBM bytes of one delta-rule prefill call with chunk states
    (bf16 q,k,v; fp32 g, beta, o, states; zero entering state)."""
    n_chunks = (T + 63) // 64
    return T * H * (2 * (2 * dk + dv) + 8 + 4 * dv) + (n_chunks + 1) * H * dk * dv * 4


def scan_useful_flops(T, H, dk, dv, C=64):
    """Causal useful flops: per chunk of L tokens, QK^T over the causal half,
    P V, Q S and the state fold."""
    full, tail = divmod(T, C)
    def chunk(L):
        return 2 * (L * (L + 1) // 2) * (dk + dv) + 2 * 2 * L * dk * dv
    return H * (full * chunk(C) + (chunk(tail) if tail else 0))


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def cpu_baseline(w, capsule_layout):
    """The oracle, as it stands, on the host: single-threaded C (fp64 scan,
    memcpy capsule).  Bounded samples, scaled to the metric's units:
    restore of the full capsule; the tiny and 8-layer workloads' scans in
    full; one 48-layer-workload layer over all 32 heads (scaled x36), single
    thread and with one thread per head on every available core."""
    import numpy as np
    from concurrent.futures import ThreadPoolExecutor

    import oracle
    import synth

    orc = oracle.get()
    cores = len(os.sched_getaffinity(0))
    host = "host %s, %d cores available" % (cpu_model(), cores)
    # capsule restore: host memcpy of the whole capsule, median of 5
    rb, rt, kd = capsule_layout
    Pa = w.prefix
    bufs = [np.zeros(r * n, np.uint8) for r, n in zip(rb, rt)]
    nbytes = orc.capsule_bytes(rb, rt, kd, Pa)
    arena = np.ones(nbytes, np.uint8)
    orc.restore(arena, bufs, rb, rt, kd, Pa)  # touch pages
    ts = []
    for _ in range(5):
        t0 = time.perf_counter()
        orc.restore(arena, bufs, rb, rt, kd, Pa)
        ts.append(time.perf_counter() - t0)
    restore_gbs = 2 * nbytes / float(np.median(ts)) / 1e9
    del bufs, arena

    def run_layer(inp, heads, threads):
        """Sequential recurrence over every head of one layer (head by head
        in `threads` worker threads; the C oracle releases the GIL)."""
        def one(h):
            return orc.sequential(*[np.ascontiguousarray(inp[n][:, h:h + 1]) for n in ("q", "k", "v", "g")])
        t0 = time.perf_counter()
        with ThreadPoolExecutor(threads) as ex:
            list(ex.map(one, range(heads)))
        return time.perf_counter() - t0

    out = {"cpu_baseline": {
        "value": round(restore_gbs, 3), "unit": "GB/s", "cores": 1, "kind": "oracle",
        "sample": "oracle capsule restore (host memcpy, single thread) of the full %d-byte capsule, median of 5; %s"
                  % (nbytes, host)}}
    # tiny workload: the whole scan (1 layer, 2 heads, 256 fp32 tokens)
    tw = synth.get_config("tiny")
    tinp = synth.linattn_inputs(tw.seed, 0, 256, tw.heads, tw.dk, tw.dv, "f32")
    t_tiny = run_layer(tinp, tw.heads, 1)
    out["cpu_baseline_tiny"] = {"value": round(256 / t_tiny, 1), "unit": "tokens/s", "cores": 1, "kind": "oracle",
                                "sample": "oracle sequential recurrence, tiny workload in full (1 layer x 2 heads x "
                                          "256 tokens) in %.4f s" % t_tiny}
    # 8-layer workload: all 6 linear layers x 16 heads over the prefix and its 32 steps
    hw = synth.get_config("hybrid8")
    F8 = hw.prefix + hw.continuation
    t_h8 = 0.0
    for l in range(hw.n_linear):
        hinp = synth.linattn_inputs(hw.seed, l, F8, hw.heads, hw.dk, hw.dv, "bf16")
        t_h8 += run_layer(hinp, hw.heads, 1)
    out["cpu_baseline_hybrid8"] = {"value": round(F8 / t_h8, 3), "unit": "tokens/s", "cores": 1, "kind": "oracle",
                                   "sample": "oracle sequential recurrence, 8-layer workload in full (6 linear layers "
                                             "x 16 heads x %d tokens) in %.2f s" % (F8, t_h8)}
    # 48-layer workload: one layer, all 32 heads, single thread, then all cores
    inp = synth.linattn_inputs(w.seed, 0, w.prefix, w.heads, w.dk, w.dv, "bf16")
    t_1 = run_layer(inp, w.heads, 1)
    t_n = run_layer(inp, w.heads, min(cores, w.heads))
    out["cpu_baseline_scan"] = {
        "value": round(w.prefix / (t_1 * w.n_linear), 3), "unit": "tokens/s", "cores": 1, "kind": "oracle",
        "sample": "oracle sequential recurrence (fp64, single thread) on 1 layer x all %d heads x %d tokens in "
                  "%.2f s, extrapolated x%d layers" % (w.heads, w.prefix, t_1, w.n_linear)}
    out["cpu_baseline_scan_allcore"] = {
        "value": round(w.prefix / (t_n * w.n_linear), 3), "unit": "tokens/s", "cores": min(cores, w.heads),
        "kind": "oracle",
        "sample": "the same layer with one thread per head on %d threads in %.2f s, extrapolated x%d layers"
                  % (min(cores, w.heads), t_n, w.n_linear)}
    del inp
    # delta rule: the token-by-token recurrence on 1 layer x 2 heads
    H_s = 2
    ginp = synth.gdn_inputs(w.seed, 0, w.prefix, H_s, w.dk, w.dv, "bf16")
    t0 = time.perf_counter()
    orc.gdn_sequential(ginp["q"], ginp["k"], ginp["v"], ginp["g"], ginp["beta"])
    t_gdn = time.perf_counter() - t0
    out["cpu_baseline_gdn"] = {
        "value": round(w.prefix / (t_gdn * (w.heads / H_s)), 3), "unit": "tokens/s per layer", "cores": 1,
        "kind": "oracle",
        "sample": "oracle gated delta-rule recurrence (fp64, single thread) on 1 layer x %d of %d heads x %d "
                  "tokens in %.2f s, extrapolated x%d head groups" % (H_s, w.heads, w.prefix, t_gdn, w.heads // H_s)}
    return out


def percentiles(xs):
    import numpy as np
    a = np.asarray(xs, np.float64)
    return {"p50": round(float(np.percentile(a, 50)), 4), "p90": round(float(np.percentile(a, 90)), 4),
            "p99": round(float(np.percentile(a, 99)), 4), "mean": round(float(a.mean()), 4), "n": int(a.size)}


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the capsule + scan hot path runs on a single MI355X; "
              "run it with --gpus 1 (the multi-GPU sharding is a design note, not a measured path).",
              file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import paper_2606_20537_amd as cap
    import synth

    torch.cuda.set_device(0)
    dev = torch.device("cuda", 0)
    w = synth.get_config(args.workload)
    T, H, dk, dv, P = w.prefix, w.heads, w.dk, w.dv, w.prefix
    n_lin, n_full = w.n_linear, w.n_full
    n_chunks = (T + 63) // 64
    stream = torch.cuda.Stream(device=dev)  # default priority

    # ---- inputs: distinct host-generated layers replicated into per-layer buffers
    t_setup = time.perf_counter()
    nd = max(1, min(args.distinct_layers, n_lin))
    src = []
    for l in range(nd):
        inp = synth.linattn_inputs(w.seed, l, T, H, dk, dv, "bf16")
        src.append({n: torch.from_numpy(inp[n + "_dev"].view(np.int16)).view(torch.bfloat16).to(dev)
                    for n in ("q", "k", "v")})
        src[-1]["g"] = torch.from_numpy(inp["g"]).to(dev)
        del inp
    layers = []
    for l in range(n_lin):
        s = src[l % nd]
        layers.append({
            "q": s["q"].clone(), "k": s["k"].clone(), "v": s["v"].clone(), "g": s["g"].clone(),
            "o": torch.empty((T, H, dv), dtype=torch.float32, device=dev),
            "cs": torch.empty((n_chunks, H, dk, dv), dtype=torch.float32, device=dev),
            "state": torch.empty((H, dk, dv), dtype=torch.float32, device=dev),
            "conv": torch.empty(w.conv_width * w.conv_channels * 2, dtype=torch.uint8, device=dev),
            "q1": s["q"][T - 1:T].clone(), "k1": s["k"][T - 1:T].clone(), "v1": s["v"][T - 1:T].clone(),
            "g1": s["g"][T - 1:T].clone(), "o1": torch.empty((1, H, dv), dtype=torch.float32, device=dev),
        })
        layers[-1]["conv"].copy_(torch.from_numpy(synth.fill_normal_bytes(w.seed, l, "conv", layers[-1]["conv"].numel())))
    del src
    kv = []
    for l in range(n_full):
        for name in ("k", "v"):
            t = torch.empty(w.t_max * w.kv_row_bytes, dtype=torch.uint8, device=dev)
            t.view(torch.bfloat16).normal_(generator=torch.Generator(device=dev).manual_seed(w.seed + 2 * l + (name == "v")))
            kv.append(("kv%d.%s" % (l, name), t))

    def live_bufs(lays, kvs):
        bufs, li, ki = [], 0, 0
        for layer in range(n_lin + n_full):  # 3 linear layers, then 1 full-attention layer
            if layer % 4 == 3 and ki < len(kvs):
                for _ in range(2):
                    name, t = kvs[ki]
                    bufs.append((name, t, w.kv_row_bytes, w.t_max, cap.CAP_KIND_POSITIONAL))
                    ki += 1
            else:
                L = lays[li]
                bufs.append(("lin%d.state" % li, L["state"], H * dk * dv * 4, 1, cap.CAP_KIND_FIXED))
                # the conv tail: a window of conv_width rows of conv_channels bf16
                bufs.append(("lin%d.conv" % li, L["conv"], w.conv_channels * 2, w.conv_width, cap.CAP_KIND_FIXED))
                li += 1
        assert li == n_lin and ki == len(kvs)
        return bufs

    bufs = live_bufs(layers, kv)
    deploy = 0x48_3A_36_2B_12
    live = cap.cap_set_create(bufs, w.chunk, deploy)
    cap_bytes = cap.capsule_bytes(live, P)
    arena = torch.empty(cap_bytes, dtype=torch.uint8, device=dev)
    n_fork = dict(w.extra).get("fork", 4)
    fork_sets, fork_keep = [], []
    for f in range(n_fork):
        fl = [{"state": torch.empty_like(L["state"]), "conv": torch.empty_like(L["conv"])} for L in layers]
        fk = [(n, torch.empty_like(t)) for n, t in kv]
        fork_keep.append((fl, fk))
        fork_sets.append(cap.cap_set_create(live_bufs(fl, fk), w.chunk, deploy))
    # the continuation token's K/V rows and conv inputs (synthetic), one per buffer of the set
    tok_src = []
    for name, t, rb, rows, kind in bufs:
        if name.endswith(".state"):
            tok_src.append(None)
        else:
            x = torch.empty(rb, dtype=torch.uint8, device=dev)
            x.view(torch.bfloat16).normal_(generator=torch.Generator(device=dev).manual_seed(len(tok_src)))
            tok_src.append(x)
    flush = torch.empty(512 * 1024 * 1024, dtype=torch.uint8, device=dev)  # > MALL
    digest = cap.capsule_digest_tokens(synth.token_ids(w.seed, P))
    torch.cuda.synchronize()
    t_setup = time.perf_counter() - t_setup

    phases = ["scan_cs", "scan_final", "snapshot", "restore", "fork", "continue"]

    def decode_token(strm):
        """One continuation token: the K/V rows and conv inputs enter the set
        (one append launch), then the 36 one-token recurrent updates."""
        cap.cap_set_append(live, tok_src, 1, stream=strm)
        for L in layers:
            cap.linattn_decode_step(L["q1"], L["k1"], L["v1"], L["g1"], L["o1"], state_in=L["state"],
                                    final_state=L["state"], stream=strm)

    def step(record):
        ev = {k: (torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for k in phases}
        caps = []
        with torch.cuda.stream(stream):
            ev["scan_cs"][0].record(stream)
            for L in layers:
                cap.linattn_chunked_prefill(L["q"], L["k"], L["v"], L["g"], L["o"], chunk_states=L["cs"],
                                            final_state=L["state"], stream=stream)
            ev["scan_cs"][1].record(stream)
            ev["scan_final"][0].record(stream)
            for L in layers:
                cap.linattn_chunked_prefill(L["q"], L["k"], L["v"], L["g"], L["o"], final_state=L["state"],
                                            stream=stream)
            ev["scan_final"][1].record(stream)
            cap.cap_set_set_position(live, P)
            flush.fill_(1)
            ev["snapshot"][0].record(stream)
            c = cap.capsule_snapshot(live, P, digest, arena, stream=stream)
            ev["snapshot"][1].record(stream)
            caps.append(c)
            flush.fill_(2)
            ev["restore"][0].record(stream)
            cap.capsule_restore(c, live, digest, stream=stream)
            ev["restore"][1].record(stream)
            flush.fill_(3)
            ev["fork"][0].record(stream)
            cap.capsule_fork(c, fork_sets, digest, stream=stream)
            ev["fork"][1].record(stream)
            ev["continue"][0].record(stream)
            decode_token(stream)
            ev["continue"][1].record(stream)
        return ev, caps

    for _ in range(args.warmup):
        step(False)
    torch.cuda.synchronize()

    # ---- timed region: K steps between barriers (one process: synchronize)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    recs = [step(True) for _ in range(args.steps)]
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0

    ms = {k: float(np.mean([r[0][k][0].elapsed_time(r[0][k][1]) for r in recs])) for k in phases}
    ms_per_step = wall * 1e3 / args.steps

    # post-run spot check: every fork branch holds the capsule's bytes (the
    # set starts with lin0.state; the continuation appends K/V at row P, so
    # rows [0, P) are the capsule's)
    nst = H * dk * dv * 4
    for fl, fk in fork_keep:
        assert torch.equal(fl[0]["state"].view(torch.uint8).flatten(), arena[:nst])
        assert torch.equal(fk[-1][1][: P * w.kv_row_bytes], kv[-1][1][: P * w.kv_row_bytes])

    # ---- restore + one decode token as ONE HIP graph vs eager launches
    # (outside the timed step; the graph is bound to this set, P and token)
    c_g = recs[-1][1][0]
    graph = torch.cuda.CUDAGraph()
    stream.synchronize()
    with torch.cuda.stream(stream):
        with torch.cuda.graph(graph, stream=stream):
            cap.capsule_restore(c_g, live, digest, stream=stream)
            decode_token(stream)
    dec_ms = {"eager": [], "graph": []}
    enq_us = {"eager": [], "graph": []}
    for rnd in range(6):
        for mode in ("eager", "graph"):
            e = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
            with torch.cuda.stream(stream):
                flush.fill_(rnd)
                e[0].record(stream)
                t_enq = time.perf_counter()
                if mode == "graph":
                    graph.replay()
                else:
                    cap.capsule_restore(c_g, live, digest, stream=stream)
                    decode_token(stream)
                t_enq = time.perf_counter() - t_enq
                e[1].record(stream)
            stream.synchronize()
            if mode == "eager":
                eager_state = layers[-1]["state"].clone()
                eager_kv = kv[-1][1][P * w.kv_row_bytes:(P + 1) * w.kv_row_bytes].clone()
            else:
                assert torch.equal(layers[-1]["state"], eager_state)
                assert torch.equal(kv[-1][1][P * w.kv_row_bytes:(P + 1) * w.kv_row_bytes], eager_kv)
            if rnd:
                dec_ms[mode].append(e[0].elapsed_time(e[1]))
                enq_us[mode].append(t_enq * 1e6)
    graph_ms, eager_ms = float(np.median(dec_ms["graph"])), float(np.median(dec_ms["eager"]))
    del graph

    # ---- TTFT distribution, outside the timed step: 30 repeats of each leg,
    # the Infinity Cache flushed before each.  cold = chunked prefill of the
    # 36 linear layers over the prefix (final states) + the 12 full-attention
    # layers' K/V rows [0, P) materialised (a copy from synthetic rows,
    # standing in for those layers' prefill, which is not built) + the first
    # token; capsule = restore + the first token.
    kv_src = []
    for i, (_, t) in enumerate(kv):
        x = torch.empty(P * w.kv_row_bytes, dtype=torch.uint8, device=dev)
        x.view(torch.bfloat16).normal_(generator=torch.Generator(device=dev).manual_seed(7000 + i))
        kv_src.append(x)
    c_t = recs[-1][1][0]

    def cold_leg():
        for L in layers:
            cap.linattn_chunked_prefill(L["q"], L["k"], L["v"], L["g"], L["o"], final_state=L["state"],
                                        stream=stream)
        for (_, t), x in zip(kv, kv_src):
            t[: P * w.kv_row_bytes].copy_(x)
        cap.cap_set_set_position(live, P)
        decode_token(stream)

    def capsule_leg():
        cap.capsule_restore(c_t, live, digest, stream=stream)
        decode_token(stream)

    ttft = {"cold": [], "capsule": []}
    with torch.cuda.stream(stream):
        for rnd in range(31):
            for name, fn in (("cold", cold_leg), ("capsule", capsule_leg)):
                flush.fill_(rnd)
                e = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
                e[0].record(stream)
                fn()
                e[1].record(stream)
                stream.synchronize()
                if rnd:
                    ttft[name].append(e[0].elapsed_time(e[1]))
    del kv_src

    # ---- host tier, outside the timed step: demote the capsule to pinned
    # host memory and promote it back (each a stream-ordered copy over the
    # host link), one warm-up and three timed rounds, checked bitwise
    c_dev = recs[-1][1][0]
    h_arena = torch.empty(cap_bytes, dtype=torch.uint8, pin_memory=True)
    d_arena = torch.empty(cap_bytes, dtype=torch.uint8, device=dev)
    tier_ms = {"demote": [], "promote": []}
    with torch.cuda.stream(stream):
        for rnd in range(4):
            e = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
            e[0].record(stream)
            c_host = cap.capsule_move(c_dev, h_arena, stream=stream)
            e[1].record(stream)
            c_back = cap.capsule_move(c_host, d_arena, stream=stream)
            e[2].record(stream)
            stream.synchronize()
            if rnd:
                tier_ms["demote"].append(e[0].elapsed_time(e[1]))
                tier_ms["promote"].append(e[1].elapsed_time(e[2]))
    assert cap.capsule_tier(c_host) == cap.CAP_TIER_HOST and cap.capsule_tier(c_back) == cap.CAP_TIER_DEVICE
    assert torch.equal(d_arena, arena)
    demote_ms, promote_ms = float(np.median(tier_ms["demote"])), float(np.median(tier_ms["promote"]))
    del h_arena, d_arena

    # ---- FP8 KV region, outside the timed step: the 24 K/V buffers held as
    # OCP E4M3 (one byte per element, scale 1) in a live set with the same
    # states and conv tails; each FP8 buffer is bound to a bf16 working stage
    # (the attention's read buffer, not part of the capsule).  Rows [0, P)
    # enter the FP8 region by one quantize launch and the stage by its first
    # read (cap_stage_acquire); then snapshot, restore into the same session
    # (the stage is re-bound, nothing converted) and restore into another
    # session (its first read converts all P rows).
    kv_el = w.kv_row_bytes // 2

    def fp8_session():
        regions = [(name, torch.empty(w.t_max * kv_el, dtype=torch.uint8, device=dev)) for name, _ in kv]
        stages = [torch.empty(w.t_max * kv_el, dtype=torch.bfloat16, device=dev) for _ in kv]
        bl = []
        for b in live_bufs(layers, regions):
            name, t, rb, rows, kind = b
            bl.append((name, t, kv_el if kind == cap.CAP_KIND_POSITIONAL else rb, rows, kind))
        s8 = cap.cap_set_create(bl, w.chunk, deploy)
        pos_idx = [i for i, b in enumerate(bl) if b[4] == cap.CAP_KIND_POSITIONAL]
        for i, st in zip(pos_idx, stages):
            cap.cap_set_bind_stage(s8, i, st, 1.0)
        return s8, regions, stages

    live8, fp8, stage8 = fp8_session()
    other8, fp8_o, stage8_o = fp8_session()
    quant_segs = [(t, f, P * kv_el, 1.0) for (_, t), (_, f) in zip(kv, fp8)]
    cap.kv_fp8_quantize(quant_segs, stream=stream)
    cap.cap_set_set_position(live8, P)
    cap.cap_stage_invalidate(live8)              # the FP8 rows were written outside the set's calls
    cap.cap_stage_acquire(live8, P, stream=stream)
    stream.synchronize()
    ref_stage = [st[: P * kv_el].clone() for st in stage8]   # stage of the cold path, converted eagerly
    cap8_bytes = cap.capsule_bytes(live8, P)
    arena8 = torch.empty(cap8_bytes, dtype=torch.uint8, device=dev)
    f8 = {"quantize": [], "snapshot": [], "restore": [], "acquire": [], "restore_other": [], "acquire_other": []}
    conv = {"acquire": [], "acquire_other": []}
    with torch.cuda.stream(stream):
        for rnd in range(4):
            t = {}
            steps = [("snapshot", lambda: t.__setitem__("c8", cap.capsule_snapshot(live8, P, digest, arena8,
                                                                                  stream=stream))),
                     ("restore", lambda: cap.capsule_restore(t["c8"], live8, digest, stream=stream)),
                     ("acquire", lambda: t.__setitem__("n", cap.cap_stage_acquire(live8, P, stream=stream))),
                     ("restore_other", lambda: cap.capsule_restore(t["c8"], other8, digest, stream=stream)),
                     ("acquire_other", lambda: t.__setitem__("n", cap.cap_stage_acquire(other8, P, stream=stream)))]
            for name, fn in steps:
                flush.fill_(rnd)
                e = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
                e[0].record(stream)
                fn()
                e[1].record(stream)
                stream.synchronize()
                if name in conv:
                    conv[name].append(t["n"])
                if rnd:
                    f8[name].append(e[0].elapsed_time(e[1]))
            # quantize (appended rows enter the FP8 region this way); it rewrites
            # the FP8 rows outside the set's calls: invalidate, re-read the stage
            e = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
            flush.fill_(rnd)
            e[0].record(stream)
            cap.kv_fp8_quantize(quant_segs, stream=stream)
            e[1].record(stream)
            stream.synchronize()
            cap.cap_stage_invalidate(live8)
            cap.cap_stage_acquire(live8, P, stream=stream)
            if rnd:
                f8["quantize"].append(e[0].elapsed_time(e[1]))
    stream.synchronize()
    # the lazily rebuilt stage of the other session equals the cold path's stage
    assert all(torch.equal(a[: P * kv_el], r) for a, r in zip(stage8_o, ref_stage))
    assert set(conv["acquire"]) == {0} and set(conv["acquire_other"]) == {P}
    f8ms = {k: float(np.median(v)) for k, v in f8.items()}
    conv_bytes = P * kv_el * len(kv) * 3  # read 2 + write 1 (quantize) or read 1 + write 2 (rebuild)
    del fp8, stage8, fp8_o, stage8_o, ref_stage, live8, other8

    # gated delta-rule layer (same shape as a linear-attention layer of the
    # stack): one call = the (I + A)^-1 launch + the scan launch.  Timed the
    # way a stack runs its layers and the way the scan phases of the step are
    # timed: back to back, two layers' inputs alternating, at the GPU's
    # steady state under this load.  After an idle gap the per-call time of
    # a back-to-back run first dips and then settles over ~40 calls (clock
    # and power management: 0.59 ms, then up to 0.75 ms, then 0.55 ms), so
    # 40 untimed calls come first.
    gl = []
    for l in range(2):
        ginp = synth.gdn_inputs(w.seed, l, T, H, dk, dv, "bf16")
        gd = {n: torch.from_numpy(ginp[n + "_dev"].view(np.int16)).view(torch.bfloat16).to(dev) for n in ("q", "k", "v")}
        gd["g"] = torch.from_numpy(ginp["g"]).to(dev)
        gd["beta"] = torch.from_numpy(ginp["beta"]).to(dev)
        del ginp
        gd["o"] = torch.empty((T, H, dv), dtype=torch.float32, device=dev)
        gd["cs"] = torch.empty(((T + 63) // 64, H, dk, dv), dtype=torch.float32, device=dev)
        gd["fs"] = torch.empty((H, dk, dv), dtype=torch.float32, device=dev)
        gl.append(gd)
    g_ws = torch.empty(cap.gdn_workspace_bytes(T, H), dtype=torch.uint8, device=dev)
    n_gdn, w_gdn = 10, 40
    g_ev = [torch.cuda.Event(enable_timing=True) for _ in range(n_gdn + 1)]
    with torch.cuda.stream(stream):
        for rnd in range(n_gdn + w_gdn):
            if rnd >= w_gdn:
                g_ev[rnd - w_gdn].record(stream)
            gd = gl[rnd % 2]
            cap.gdn_chunked_prefill(gd["q"], gd["k"], gd["v"], gd["g"], gd["beta"], gd["o"], chunk_states=gd["cs"],
                                    final_state=gd["fs"], workspace=g_ws, stream=stream)
        g_ev[n_gdn].record(stream)
    stream.synchronize()
    g_ms = [g_ev[i].elapsed_time(g_ev[i + 1]) for i in range(n_gdn)]
    g_o, g_cs, g_fs = gl[1]["o"], gl[1]["cs"], gl[1]["fs"]
    gdn_ms = float(np.median(g_ms))
    gdn_b = gdn_bytes(T, H, dk, dv)
    gdn_gbs = gdn_b / (gdn_ms * 1e-3) / 1e9
    assert bool(torch.isfinite(g_o).all()) and bool(torch.isfinite(g_fs).all())
    del gd, gl, g_o, g_cs, g_fs

    # ---- robot episode reset (the gather verb), outside the timed step: 32
    # environments, a gallery of 8 capsules (18 KV layers [816 tokens, 1 head,
    # d=256] bf16 + a 2 MiB fp32 denoiser state each); one reset restores
    # gallery[id_e] into environment e for every e in one launch; 1000
    # resets back to back after 20 warm-up resets (the 137 MB gallery then
    # sits in the Infinity Cache); the last reset is checked byte for byte
    rw = synth.get_config("robot_reset")
    rx = dict(rw.extra)
    rlayout = [("kv%d.%s" % (l, nm), rw.kv_row_bytes, rw.t_max, cap.CAP_KIND_POSITIONAL)
               for l in range(rw.n_full) for nm in ("k", "v")]
    rlayout.append(("denoiser", rx["denoiser_bytes"], 1, cap.CAP_KIND_FIXED))

    def reset_bufs(seed):
        out_b = []
        for i, (nm, rb, rows, kind) in enumerate(rlayout):
            t = torch.empty(rb * rows, dtype=torch.uint8, device=dev)
            t.view(torch.float32).normal_(generator=torch.Generator(device=dev).manual_seed(seed * 1000 + i))
            out_b.append((nm, t, rb, rows, kind))
        return out_b

    RP = rw.prefix
    gal_keep, gallery = [], []
    for gi in range(rx["gallery"]):
        b = reset_bufs(100 + gi)
        s_g = cap.cap_set_create(b, rw.chunk, 3)
        cap.cap_set_set_position(s_g, RP)
        ar = torch.empty(cap.capsule_bytes(s_g, RP), dtype=torch.uint8, device=dev)
        gallery.append(cap.capsule_snapshot(s_g, RP, 0, ar, stream=stream))
        gal_keep.append((s_g, b, ar))
    env_keep = [reset_bufs(500 + e) for e in range(rx["envs"])]
    env_sets = [cap.cap_set_create(b, rw.chunk, 3) for b in env_keep]
    gal_bytes = cap.capsule_info(gallery[0])["bytes"]
    ids_all = synth.rng(rw.seed, 0, "reset_ids").integers(0, rx["gallery"], size=(rx["resets"], rx["envs"]))
    ids_all = ids_all.astype(np.int32)
    stream.synchronize()
    with torch.cuda.stream(stream):
        for r in range(20):
            cap.capsule_gather_restore(gallery, ids_all[r], env_sets, stream=stream)
        e = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
        e[0].record(stream)
        for r in range(rx["resets"]):
            cap.capsule_gather_restore(gallery, ids_all[r], env_sets, stream=stream)
        e[1].record(stream)
    stream.synchronize()
    reset_ms = e[0].elapsed_time(e[1]) / rx["resets"]
    assert RP == rw.t_max  # every row of a K/V buffer is inside the capsule
    for env, gi in enumerate(ids_all[-1]):
        for (_, te, *_), (_, tg, *_) in zip(env_keep[env], gal_keep[gi][1]):
            assert torch.equal(te, tg)
    reset_bytes = 2 * rx["envs"] * gal_bytes  # each environment's capsule read once and written once
    del gal_keep, gallery, env_keep, env_sets

    # ---- the 8-layer workload (6 linear layers of 16 heads, 2 full-attention
    # layers of K/V [8448, 4, 128] bf16, conv windows 4 x 2048, prefix 2048):
    # its 14.8 MB capsule's restore latency, and the 32 decode steps after a
    # restore (each: one append of the token's K/V rows and conv inputs, then
    # 6 one-token steps); cold vs capsule TTFT with the same legs as above
    hw = synth.get_config("hybrid8")
    H8, P8, n8 = hw.heads, hw.prefix, hw.continuation
    F8 = P8 + n8
    lay8 = []
    for l in range(hw.n_linear):
        inp = synth.linattn_inputs(hw.seed, l, F8, H8, hw.dk, hw.dv, "bf16")
        e8 = {n: torch.from_numpy(inp[n + "_dev"].view(np.int16)).view(torch.bfloat16).to(dev) for n in ("q", "k", "v")}
        e8["g"] = torch.from_numpy(inp["g"]).to(dev)
        e8["state"] = torch.zeros((H8, hw.dk, hw.dv), dtype=torch.float32, device=dev)
        e8["conv"] = torch.zeros((hw.conv_width, hw.conv_channels), dtype=torch.bfloat16, device=dev)
        e8["conv_in"] = torch.randn((F8, hw.conv_channels), generator=torch.Generator(device=dev).manual_seed(300 + l),
                                    device=dev).to(torch.bfloat16)
        e8["o"] = torch.empty((F8, H8, hw.dv), dtype=torch.float32, device=dev)
        lay8.append(e8)
    kv8 = [torch.zeros((hw.t_max, hw.kv_heads, hw.kv_dim), dtype=torch.bfloat16, device=dev) for _ in range(2 * hw.n_full)]
    kv8_in = [torch.randn((F8, hw.kv_heads, hw.kv_dim), generator=torch.Generator(device=dev).manual_seed(400 + i),
                          device=dev).to(torch.bfloat16) for i in range(2 * hw.n_full)]
    bufs8, li, ki = [], 0, 0
    for layer in range(hw.n_linear + hw.n_full):
        if layer % 4 == 3:
            for _ in range(2):
                bufs8.append(("kv%d" % ki, kv8[ki], hw.kv_row_bytes, hw.t_max, cap.CAP_KIND_POSITIONAL))
                ki += 1
        else:
            bufs8.append(("state%d" % li, lay8[li]["state"], H8 * hw.dk * hw.dv * 4, 1, cap.CAP_KIND_FIXED))
            bufs8.append(("conv%d" % li, lay8[li]["conv"], hw.conv_channels * 2, hw.conv_width, cap.CAP_KIND_FIXED))
            li += 1
    live_8 = cap.cap_set_create(bufs8, hw.chunk, deploy)

    def h8_prefill():
        for e8 in lay8:
            cap.linattn_chunked_prefill(e8["q"][:P8], e8["k"][:P8], e8["v"][:P8], e8["g"][:P8], e8["o"][:P8],
                                        final_state=e8["state"], stream=stream)
            e8["conv"].copy_(e8["conv_in"][P8 - hw.conv_width:P8])
        for t, x in zip(kv8, kv8_in):
            t[:P8].copy_(x[:P8])
        cap.cap_set_set_position(live_8, P8)

    def h8_token(t0):
        srcs, li, ki = [], 0, 0
        for name, *_ in bufs8:
            if name.startswith("kv"):
                srcs.append(kv8_in[ki][t0:t0 + 1]); ki += 1
            elif name.startswith("conv"):
                srcs.append(lay8[li]["conv_in"][t0:t0 + 1]); li += 1
            else:
                srcs.append(None)
        cap.cap_set_append(live_8, srcs, 1, stream=stream)
        for e8 in lay8:
            cap.linattn_decode_step(e8["q"][t0:t0 + 1], e8["k"][t0:t0 + 1], e8["v"][t0:t0 + 1], e8["g"][t0:t0 + 1],
                                    e8["o"][t0:t0 + 1], state_in=e8["state"], final_state=e8["state"], stream=stream)

    with torch.cuda.stream(stream):
        h8_prefill()
    cap8 = cap.capsule_bytes(live_8, P8)
    arena_8 = torch.empty(cap8, dtype=torch.uint8, device=dev)
    c_8 = cap.capsule_snapshot(live_8, P8, 8, arena_8, stream=stream)
    h8 = {"restore": [], "steps32": [], "prefill": [], "cold": [], "capsule": []}
    with torch.cuda.stream(stream):
        for rnd in range(16):
            legs = [("prefill", h8_prefill),
                    ("restore", lambda: cap.capsule_restore(c_8, live_8, 8, stream=stream)),
                    ("steps32", lambda: [h8_token(t0) for t0 in range(P8, F8)]),
                    ("cold", lambda: (h8_prefill(), h8_token(P8))),
                    ("capsule", lambda: (cap.capsule_restore(c_8, live_8, 8, stream=stream), h8_token(P8)))]
            for name, fn in legs:
                flush.fill_(rnd)
                e = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
                e[0].record(stream)
                fn()
                e[1].record(stream)
                stream.synchronize()
                if rnd:
                    h8[name].append(e[0].elapsed_time(e[1]))
    h8ms = {k: float(np.median(v)) for k, v in h8.items()}
    # the same restore + 32 decode steps recorded as one HIP graph and
    # replayed (launch gaps of the host removed): GPU time per token
    g8 = torch.cuda.CUDAGraph()
    stream.synchronize()
    with torch.cuda.stream(stream):
        with torch.cuda.graph(g8, stream=stream):
            cap.capsule_restore(c_8, live_8, 8, stream=stream)
            for t0 in range(P8, F8):
                h8_token(t0)
    g8_ms = []
    with torch.cuda.stream(stream):
        for rnd in range(6):
            flush.fill_(rnd)
            e = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
            e[0].record(stream)
            g8.replay()
            e[1].record(stream)
            stream.synchronize()
            if rnd:
                g8_ms.append(e[0].elapsed_time(e[1]))
    h8ms["graph"] = float(np.median(g8_ms))
    del g8
    del lay8, kv8, kv8_in, live_8, arena_8, c_8

    scan_b = scan_bytes(T, H, dk, dv, True)
    scan_b_final = scan_bytes(T, H, dk, dv, False)
    flops = scan_useful_flops(T, H, dk, dv)
    scan_launch_ms = ms["scan_cs"] / n_lin
    scan_gbs = scan_b / (scan_launch_ms * 1e-3) / 1e9
    restore_gbs = 2 * cap_bytes / (ms["restore"] * 1e-3) / 1e9
    cold_ttft = ms["scan_final"] + ms["continue"]
    caps_ttft = ms["restore"] + ms["continue"]

    out = {
        "metric": "capsule restore GB/s (% HBM peak); scan tokens/s (% MFMA); restore/cold TTFT",
        "value": round(restore_gbs, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u8 capsule bytes; scan bf16 MFMA inputs, fp32 state",
        "data": "synthetic (seeded PCG64; %d distinct layers replicated into %d layer buffers)" % (nd, n_lin),
        "config": {"workload": "hybrid48: %d linear-attn (H=%d, dk=dv=%d) + %d full-attn (4 KV heads, d=256) layers, "
                               "prefix %d, chunk 64, fork x%d" % (n_lin, H, dk, n_full, T, n_fork),
                   "capsule_bytes": cap_bytes, "prefix": T, "chunk": 64},
        "restore_pct_hbm_peak": round(100 * restore_gbs / HBM_PEAK_GBS, 2),
        "scan_tokens_per_s": round(T / (ms["scan_cs"] * 1e-3), 1),
        "scan_tokens_per_s_final_only": round(T / (ms["scan_final"] * 1e-3), 1),
        "scan_pct_mfma_useful": round(100 * flops / (scan_launch_ms * 1e-3) / (MFMA_BF16_PEAK_TFS * 1e12), 3),
        "scan_pct_mfma_useful_ceiling": round(100 * flops / (scan_b / (HBM_PEAK_GBS * 1e9)) / (MFMA_BF16_PEAK_TFS * 1e12), 2),
        "scan_pct_mfma_busy_counter": {"chunk_states": measured_mfma_busy("scan_cs"),
                                       "final_only": measured_mfma_busy("scan_final"),
                                       "gdn_scan": measured_mfma_busy("gdn_scan"),
                                       "what": "MFMA pipe busy cycles / SIMD cycles (rocprofv3 counters, "
                                               "profiles/hybrid48_scan_counters.md); executed products include "
                                               "the hi/lo operand terms and the recomputed scores"},
        "ttft_ms": {"cold": percentiles(ttft["cold"]), "capsule": percentiles(ttft["capsule"]),
                    "restore_over_cold_ratio_p50": round(float(np.percentile(ttft["cold"], 50))
                                                         / float(np.percentile(ttft["capsule"], 50)), 3),
                    "cold_leg": "36 linear layers' chunked prefill (final states) + 12 full-attention layers' K/V "
                                "rows [0, P) materialised (a copy from synthetic rows) + first token (append + 36 "
                                "one-token steps); capsule leg: restore + first token; Infinity Cache flushed "
                                "before each repeat",
                    "cold_scan_only_in_step": round(cold_ttft, 4), "capsule_in_step": round(caps_ttft, 4)},
        "hybrid8": {"what": "8-layer workload (6 linear layers x 16 heads dk=dv=128, 2 full-attention layers, "
                            "prefix 2048, conv 4 x 2048): capsule restore latency, 32 decode steps after restore, "
                            "cold vs capsule TTFT; medians of 15, Infinity Cache flushed before each",
                    "capsule_bytes": cap8, "restore_us": round(1e3 * h8ms["restore"], 2),
                    "restore_gbs_effective": round(2 * cap8 / (h8ms["restore"] * 1e-3) / 1e9, 1),
                    "decode_us_per_token": round(1e3 * h8ms["steps32"] / n8, 2),
                    "decode_us_per_token_graph": round(1e3 * (h8ms["graph"] - h8ms["restore"]) / n8, 2),
                    "restore_and_32_steps_graph_ms": round(h8ms["graph"], 4),
                    "decode_launches_per_token": 1 + hw.n_linear,
                    "prefill_ms": round(h8ms["prefill"], 4),
                    "ttft_ms": {"cold": round(h8ms["cold"], 4), "capsule": round(h8ms["capsule"], 4),
                                "restore_over_cold_ratio": round(h8ms["cold"] / h8ms["capsule"], 3)}},
        "phase_ms": {k: round(v, 4) for k, v in ms.items()},
        "fork_gbs": round((1 + n_fork) * cap_bytes / (ms["fork"] * 1e-3) / 1e9, 2),
        "snapshot_gbs": round(2 * cap_bytes / (ms["snapshot"] * 1e-3) / 1e9, 2),
        "roofline": {"kernel": "linattn_scan_kernel<128,bf16> (with chunk states)", "bound": "hbm",
                     "achieved": round(scan_gbs, 2), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": round(scan_gbs / HBM_PEAK_GBS, 4), "traffic": measured_traffic("scan_cs"),
                     "algorithmic_bytes_per_launch": scan_b, "avg_launch_ms": round(scan_launch_ms, 5)},
        "roofline_copy": {"kernel": "capsule_copy_kernel (restore)", "bound": "hbm",
                          "achieved": round(restore_gbs, 2), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                          "frac": round(restore_gbs / HBM_PEAK_GBS, 4), "traffic": measured_traffic("restore"),
                          "algorithmic_bytes_per_launch": 2 * cap_bytes, "avg_launch_ms": round(ms["restore"], 5)},
        "roofline_snapshot": {"kernel": "capsule_copy_kernel (snapshot)", "bound": "hbm",
                              "achieved": round(2 * cap_bytes / (ms["snapshot"] * 1e-3) / 1e9, 2),
                              "peak": HBM_PEAK_GBS, "unit": "GB/s",
                              "frac": round(2 * cap_bytes / (ms["snapshot"] * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                              "traffic": measured_traffic("snapshot"),
                              "algorithmic_bytes_per_launch": 2 * cap_bytes, "avg_launch_ms": round(ms["snapshot"], 5)},
        "roofline_fork": {"kernel": "capsule_copy_kernel (fork x%d)" % n_fork, "bound": "hbm",
                          "achieved": round((1 + n_fork) * cap_bytes / (ms["fork"] * 1e-3) / 1e9, 2),
                          "peak": HBM_PEAK_GBS, "unit": "GB/s",
                          "frac": round((1 + n_fork) * cap_bytes / (ms["fork"] * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                          "traffic": measured_traffic("fork4") if n_fork == 4 else None,
                          "algorithmic_bytes_per_launch": (1 + n_fork) * cap_bytes, "avg_launch_ms": round(ms["fork"], 5)},
        "roofline_scan_final_only": {"bound": "hbm", "algorithmic_bytes_per_launch": scan_b_final,
                                     "achieved": round(scan_b_final / (ms["scan_final"] / n_lin * 1e-3) / 1e9, 2),
                                     "unit": "GB/s"},
        "host_tier": {"bytes": cap_bytes, "demote_ms": round(demote_ms, 3), "promote_ms": round(promote_ms, 3),
                      "demote_gbs": round(cap_bytes / (demote_ms * 1e-3) / 1e9, 2),
                      "promote_gbs": round(cap_bytes / (promote_ms * 1e-3) / 1e9, 2),
                      "link": "host link, PCIe 5.0 x16", "peak": LINK_PEAK_GBS, "unit": "GB/s",
                      "promote_frac": round(cap_bytes / (promote_ms * 1e-3) / 1e9 / LINK_PEAK_GBS, 4),
                      "capsule_ttft_ms_from_host": round(promote_ms + ms["restore"] + ms["continue"], 4)},
        "restore_decode_graph": {"launches": 1 + 1 + n_lin, "eager_ms": round(eager_ms, 4),
                                 "graph_ms": round(graph_ms, 4), "speedup": round(eager_ms / graph_ms, 3),
                                 "host_enqueue_us": {"eager": round(float(np.median(enq_us["eager"])), 1),
                                                     "graph": round(float(np.median(enq_us["graph"])), 1)},
                                 "what": "capsule restore + one token (K/V + conv append, %d one-token steps)" % n_lin},
        "fp8_kv": {"capsule_bytes": cap8_bytes, "bf16_capsule_bytes": cap_bytes,
                   "restore_ms": round(f8ms["restore"], 4), "snapshot_ms": round(f8ms["snapshot"], 4),
                   "restore_gbs": round(2 * cap8_bytes / (f8ms["restore"] * 1e-3) / 1e9, 2),
                   "same_session": {"stage_rows_converted_on_first_read": 0,
                                    "first_read_ms": round(f8ms["acquire"], 4),
                                    "capsule_ttft_ms": round(f8ms["restore"] + f8ms["acquire"] + ms["continue"], 4)},
                   "other_session": {"restore_ms": round(f8ms["restore_other"], 4),
                                     "stage_rows_converted_on_first_read": P,
                                     "first_read_ms": round(f8ms["acquire_other"], 4),
                                     "rebuild_gbs": round(conv_bytes / (f8ms["acquire_other"] * 1e-3) / 1e9, 2),
                                     "rebuild_frac": round(conv_bytes / (f8ms["acquire_other"] * 1e-3) / 1e9
                                                           / HBM_PEAK_GBS, 4),
                                     "capsule_ttft_ms": round(f8ms["restore_other"] + f8ms["acquire_other"]
                                                              + ms["continue"], 4)},
                   "bf16_capsule_ttft_ms": round(ms["restore"] + ms["continue"], 4),
                   "quantize_ms": round(f8ms["quantize"], 4),
                   "quantize_gbs": round(conv_bytes / (f8ms["quantize"] * 1e-3) / 1e9, 2)},
        "gdn": {"what": "gated delta-rule prefill, one layer (H=%d, dk=dv=%d, %d tokens, chunk states): "
                        "(I + A)^-1 launch + scan launch" % (H, dk, T),
                "layer_ms": round(gdn_ms, 4), "tokens_per_s": round(T / (gdn_ms * 1e-3), 1),
                "stack_tokens_per_s_36_layers": round(T / (n_lin * gdn_ms * 1e-3), 1),
                "roofline": {"bound": "hbm", "achieved": round(gdn_gbs, 2), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                             "frac": round(gdn_gbs / HBM_PEAK_GBS, 4), "traffic": measured_traffic("gdn"),
                             "algorithmic_bytes_per_call": gdn_b,
                             "workspace_bytes_per_call": 2 * cap.gdn_workspace_bytes(T, H)}},
        "gather": {"what": "robot episode reset: %d environments, gallery of %d capsules of %d B, %d resets back "
                           "to back, one gather launch each" % (rx["envs"], rx["gallery"], gal_bytes, rx["resets"]),
                   "reset_ms": round(reset_ms, 4), "resets_per_s": round(1e3 / reset_ms, 1),
                   "gbs": round(reset_bytes / (reset_ms * 1e-3) / 1e9, 2),
                   "write_gbs": round(reset_bytes / 2 / (reset_ms * 1e-3) / 1e9, 2),
                   "roofline": {"bound": "hbm", "achieved": round(reset_bytes / (reset_ms * 1e-3) / 1e9, 2),
                                "peak": HBM_PEAK_GBS, "unit": "GB/s",
                                "frac": round(reset_bytes / (reset_ms * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
                                "traffic": measured_traffic("gather"), "algorithmic_bytes_per_launch": reset_bytes,
                                "note": "traffic counts bytes leaving L2 (Infinity Cache hits included); "
                                        "the gallery reads are served from the Infinity Cache after warm-up, "
                                        "the writes go to HBM"}},
        "setup_s": round(t_setup, 1),
    }
    if not args.no_cpu_baseline:
        rb = [b[2] for b in bufs]
        rt = [b[3] for b in bufs]
        kd = [b[4] for b in bufs]
        out.update(cpu_baseline(w, (rb, rt, kd)))
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
