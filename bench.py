"""Benchmark: MoE-layer forward + backward throughput on one MI355X.

One step = one pass of the whole hot path over one batch: gate + top-k,
capacity-bounded dispatch, grouped-GEMM experts, combine (forward), then
combine backward, expert backward (dgrad + wgrad), dispatch backward and gate
backward, through flowmoe_layer_fwd / flowmoe_layer_bwd on two HIP streams.

Workload (default): the large-expert MoE layer, one GPU's share of a
Mixtral-shaped layer: T = 16384 tokens, M = 4096, H = 14336, E = 8 local
experts, top-2, capacity factor 1.25, SwiGLU experts, bf16 storage with fp32
accumulation, one chunk (R = 1), packed dispatch layout. Inputs are seeded
synthetic tensors already resident in HBM.

Prints one JSON line with tokens/s, the grouped-GEMM roofline (algorithmic
FLOPs per launch over the average launch time, from HIP events recorded
around every GEMM launch of the timed steps) and the fp64 CPU oracle timed on
a bounded token sample of the same inputs (whole steps for the small layers).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E
WORKLOAD = "large"


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", default=WORKLOAD,
                    help="large (default) | balanced | skewed | fine | tiny")
    ap.add_argument("--layout", default="packed")
    ap.add_argument("--gate", default="renorm", choices=("renorm", "full"),
                    help="gate weights: softmax over the k selected (renorm) or the selected "
                         "experts' full-softmax probabilities (full, Switch-style)")
    ap.add_argument("--R", type=int, default=None, help="override the chunk count")
    ap.add_argument("--expert-bias", action="store_true",
                    help="biased experts (b1, b3 on the first layer, b2 on the second)")
    ap.add_argument("--mha", action="store_true",
                    help="AT_r includes the block's multi-head attention (the workload's "
                         "sequences and heads): one step is attention + MoE layer, fwd + bwd")
    for dim, typ in (("T", int), ("M", int), ("H", int), ("E", int), ("k", int), ("f", float)):
        ap.add_argument(f"--{dim}", type=typ, default=None, help=f"override the workload's {dim}")
    ap.add_argument("--one-stream", action="store_true", help="serial schedule on one stream")
    ap.add_argument("--tile-order", default="auto", choices=("auto", "split", "joined"),
                    help="grouped-GEMM row-tile order (light tiles after every heavy one, or "
                         "walked with their expert's heavy ones)")
    ap.add_argument("--tiles", default="auto", choices=("auto", "wide", "narrow"),
                    help="grouped-GEMM tile shape")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-memory-bound", action="store_true",
                    help="skip the per-call timing of the memory-bound steps")
    ap.add_argument("--copy-probe", type=int, default=0, metavar="MIB",
                    help="after the timed steps, copy a MIB-sized buffer once: the plain copy "
                         "kernel of known size that calibrates HBM byte counters")
    return ap.parse_args()


def gemm_flops(cfg, kind: str, rows: float) -> float:
    """Algorithmic FLOPs of one grouped-GEMM launch of `kind` over `rows` kept
    rows: every expert GEMM multiplies those rows by an M x H (or H x M)
    weight, 2 * rows * M * H; SwiGLU's fused W1|W3 forward, its [dW1 | dW3]
    weight gradient and its K = 2H dgrad do twice that. The row-mode launches
    (ffn1, ffn2, dgrad1, dgrad2) cover one chunk's rows; the two weight-gradient
    launches reduce over the rows of all R chunks at once."""
    two = 2.0 if cfg.act == "swiglu" else 1.0
    mult = {"ffn1": two, "ffn2": 1.0, "dgrad1": 1.0, "dgrad2": two, "wgrad2": 1.0, "wgrad1": two}
    return 2.0 * rows * cfg.M * cfg.H * mult[kind]


def gemm_flops_per_step(cfg, kept: int) -> float:
    """All expert-GEMM FLOPs of one fwd+bwd step: 12 M H (GELU) or 18 M H
    (SwiGLU) per kept row."""
    return (18.0 if cfg.act == "swiglu" else 12.0) * kept * cfg.M * cfg.H


def attention_flops(cfg, R: int) -> dict:
    """Algorithmic FLOPs of the attention part of one step (all R chunks):
    the core per (sequence, head) is 2 d FLOPs per visible (query, key) pair
    for each of Q K^T and P V forward, and for each of the backward's five
    products (S recomputed, dP, dV, dK, dQ): N^2 pairs, or N (N + 1) / 2 when
    causal; the projections: [Q|K|V] = I W_qkv (2 T M 3M), I' = A W^O
    (2 T M^2), their two dgrads and two weight gradients (the same again
    each)."""
    T, M, N, d = cfg.T, cfg.M, cfg.seq_len, cfg.head_dim
    pairs = N * (N + 1) / 2 if cfg.causal else float(N * N)
    units = pairs * d * 2.0 * cfg.heads * (T // N)
    proj = 2.0 * T * M * 4 * M
    return {"core_fwd": 2 * units, "core_bwd": 5 * units, "proj_fwd": proj,
            "proj_dgrad": proj, "proj_wgrad": proj}


def oracle_sample_tokens(cfg, R: int) -> int:
    """Tokens of the CPU oracle's sample: the whole batch when one fp64 step
    is cheap, else the largest power-of-two number of tokens (a multiple of
    R) whose expert FLOPs stay under 6e11, so that the sample takes seconds,
    not minutes, of host time (the large layer's 1024 tokens took 191 s on
    8 cores: its numpy backward runs near 35 GFLOP/s)."""
    per_token = 2.0 * cfg.k * cfg.M * cfg.H * (9.0 if cfg.act == "swiglu" else 6.0)
    t = cfg.T
    while t > R and t * per_token > 6e11:
        t //= 2
    return max(R, (t // R) * R)


def schedule_overlap(layer, R, sc, sm, torch, mha=False):
    """One untraced-throughput step with the layer's task events (the trace
    of flowmoe_layer_fwd / flowmoe_layer_bwd: start and end of every task of
    every chunk, on the stream it runs on): each pass's span, the time each
    stream spends in its tasks, and the time both streams run a task at once
    (the overlap the two-stream schedule of Eqs. 3-6 achieves on one GPU).
    Forward: compute stream = gating, experts; comm stream = dispatch,
    combine. Backward: compute stream = experts bwd and the weight
    gradients (and with the attention, its backward per chunk and its
    weight gradients); comm stream = combine bwd, gate gradients, dispatch
    bwd."""
    from paper_2510_00207_amd import _lib as L
    def events(n):
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(n)]
        for e in ev:  # (torch creates an event's handle at its first record)
            e.record(sc)
        return ev

    fwd, bwd, (t0,) = events(8 * R), events(L.bwd_trace_len(R, mha)), events(1)
    torch.cuda.synchronize()
    t0.record(sc)
    layer.forward(sc, sm, trace=fwd)
    layer.backward(sc, sm, trace=bwd)
    torch.cuda.synchronize()
    out = {}
    for label, ev, comp in (("fwd", fwd, (0, 2)), ("bwd", bwd, (1, 4))):
        spans = {}
        for task in range(5 if label == "bwd" else 4):
            for r in range(1 if task == 4 else R):
                i = 2 * (task * R + r)
                spans[(task, r)] = (t0.elapsed_time(ev[i]), t0.elapsed_time(ev[i + 1]))
        if label == "bwd" and mha:  # (task 5: attention backward per chunk, 6: its wgrad)
            for r in range(R):
                i = 8 * R + 2 + 2 * r
                spans[(5, r)] = (t0.elapsed_time(ev[i]), t0.elapsed_time(ev[i + 1]))
            spans[(6, 0)] = (t0.elapsed_time(ev[10 * R + 2]), t0.elapsed_time(ev[10 * R + 3]))
            comp = comp + (5, 6)
        c = [v for (task, _), v in spans.items() if task in comp]
        m = [v for (task, _), v in spans.items() if task not in comp]
        # the tasks of one stream never overlap each other (stream order)
        both = sum(max(0.0, min(a1, b1) - max(a0, b0)) for a0, a1 in c for b0, b1 in m)
        lo = min(a for a, _ in spans.values())
        hi = max(b for _, b in spans.values())
        busy_c = sum(b - a for a, b in c)
        busy_m = sum(b - a for a, b in m)
        out[label] = {"span_ms": round(hi - lo, 4), "compute_stream_ms": round(busy_c, 4),
                      "comm_stream_ms": round(busy_m, 4), "overlap_ms": round(both, 4),
                      "overlap_frac_of_comm": round(both / busy_m, 4) if busy_m > 0 else None}
    return out


def widen_f64(a):
    """A stored tensor widened exactly to float64 (moe_inputs.as_f64), in
    blocks on the host's cores (the large layer's weights are 1.4e9
    elements)."""
    import concurrent.futures as cf

    import numpy as np
    from moe_inputs import as_f64
    flat = a.reshape(-1)
    out = np.empty(flat.shape[0], dtype=np.float64)
    blk = 1 << 24

    def one(lo):
        out[lo:lo + blk] = as_f64(flat[lo:lo + blk])

    with cf.ThreadPoolExecutor(max(1, min(16, len(os.sched_getaffinity(0))))) as ex:
        list(ex.map(one, range(0, flat.shape[0], blk)))
    return out.reshape(a.shape)


def memory_bound(L, layer, cfg, torch, reps: int = 20, flush=None):
    """Achieved bandwidth of the memory-bound steps of chunk 0: each C-ABI call
    repeated `reps` times back to back on one stream (inputs warm: after the
    timed steps, and small enough here to stay in the 256 MB Infinity Cache),
    against the algorithmic bytes of the step (kept rows A of the chunk):
      gate T*M*b; dispatch (scan + gather) (T + A)*M*b; combine (A + T)*M*b;
      combine bwd (T + 2A)*M*b; dispatch bwd (A + T)*M*b; gate bwd T*M*b, except
      for one selected expert under the renormalised gate, whose gradient is
      exactly zero: then the d_logits and dW_g written, (T + M)*E*4.
    With a `flush` buffer (int64, >= 512 MiB) each step is also timed with
    cold caches (the *_flushed figures)."""
    s = layer.shape
    T, M, E, k = s.T, s.M, s.E, s.k
    b = 2 if layer.dt == L.BF16 else 4
    A = int(layer.counts[0].sum().item())
    st = torch.cuda.Stream()
    x, y, dy, dx = layer.x[:T], layer.y[:T], layer.dy[:T], layer.dx[:T]
    lg, idx, w = layer.logits[:T], layer.topk_idx[:T], layer.topk_w[:T]
    dw, dl, slot = layer.d_topk_w[:T], layer.d_logits[:T], layer.slot[:T]
    cnt, off, rs, ld = layer.counts[0], layer.offsets[0], layer.row_src[0], layer.load[0]
    xd, yd, dyd, dxd = layer.x_disp[0], layer.y_disp[0], layer.dy_disp[0], layer.dx_disp[0]
    zero_gate = k == 1 and cfg.gate != "full"
    steps = {
        "gate": (lambda: L.flowmoe_gate_topk(s, x, layer.w_gate, layer.bias, lg, idx, w, stream=st),
                 T * M * b),
        "dispatch (scan + gather)": (
            lambda: L.flowmoe_dispatch(s, idx, x, cnt, off, slot, rs, ld, xd, layer.ws,
                                       layer.ws_bytes, stream=st),
            (T + A) * M * b),
        "combine": (lambda: L.flowmoe_combine(s, yd, slot, w, y, stream=st), (A + T) * M * b),
        "combine bwd": (lambda: L.flowmoe_combine_bwd(s, dy, yd, slot, w, cnt, off, dyd, dw,
                                                      stream=st), (T + 2 * A) * M * b),
        "dispatch bwd": (lambda: L.flowmoe_dispatch_bwd(s, dxd, slot, dx, stream=st),
                         (A + T) * M * b),
        "gate bwd (d_logits, dW_g)": (
            lambda: L.flowmoe_gate_topk_bwd(s, x, layer.w_gate, lg, idx, w, dw, dl, layer.dw_gate,
                                            layer.dbias, None, 0, layer.ws, layer.ws_bytes,
                                            stream=st),
            (T + M) * E * 4 if zero_gate else T * M * b),
    }
    out = {}
    flush_sum = torch.zeros((), dtype=torch.int64, device=x.device)
    for name, (fn, nbytes) in steps.items():
        fn()
        fn()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(st)
        for _ in range(reps):
            fn()
        e1.record(st)
        e1.synchronize()
        us = e0.elapsed_time(e1) / reps * 1e3
        gbs = nbytes / (us * 1e-6) / 1e9
        out[name] = {"bytes": nbytes, "us": round(us, 2), "GBps": round(gbs, 1),
                     "frac": round(gbs / PEAK_HBM_GBS, 4)}
        if flush is not None:
            # cold caches: reading a 512 MiB buffer before every call evicts
            # the inputs from L2 and the Infinity Cache and leaves only clean
            # lines behind (a fill would leave dirty lines whose write-back
            # the measured call would pay for); the call's time is that of
            # (read + call) minus that of the read alone, both back to back
            def span(with_call):
                f0, f1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                with torch.cuda.stream(st):
                    f0.record(st)
                    for _ in range(reps):
                        flush_sum.copy_(flush.sum())
                        if with_call:
                            fn()
                    f1.record(st)
                f1.synchronize()
                return f0.elapsed_time(f1) / reps * 1e3
            span(True)
            cold = span(True) - span(False)
            cgbs = nbytes / (cold * 1e-6) / 1e9
            out[name].update({"us_flushed": round(cold, 2), "GBps_flushed": round(cgbs, 1),
                              "frac_flushed": round(cgbs / PEAK_HBM_GBS, 4)})
    return out


def main():
    a = parse()
    if a.gpus != 1:
        print(f"bench.py measures one GPU only (got --gpus {a.gpus}); the multi-GPU expert-parallel "
              "path (all-to-all over RCCL) is not implemented", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from moe_inputs import get_config, make_inputs, to_torch
    from paper_2510_00207_amd import _lib as L
    from paper_2510_00207_amd.hiprt import EventArray
    from paper_2510_00207_amd.layer import MoELayer

    if not os.path.exists(L.LIB_PATH):
        from paper_2510_00207_amd import build
        build.build(verbose=False)
    L.load()
    L.flowmoe_set_gemm_tiles(a.tiles)
    L.flowmoe_set_tile_order(a.tile_order)
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")

    over = {d: getattr(a, d) for d in ("T", "M", "H", "E", "k", "f") if getattr(a, d) is not None}
    cfg = get_config(a.workload, gate=a.gate, expert_bias=a.expert_bias, mha=a.mha, **over)
    if over:  # another shape: named apart (no counter summary of the workload applies to it)
        cfg = cfg.replace(name=cfg.name + "(" + " ".join(f"{d}={v}" for d, v in over.items()) + ")")
    R = cfg.R if a.R is None else a.R
    inp = make_inputs(cfg)
    layer = MoELayer(T_total=cfg.T, M=cfg.M, H=cfg.H, E=cfg.E, k=cfg.k, R=R, f=cfg.f, act=cfg.act,
                     dtype=cfg.dtype, layout=a.layout, bias=cfg.zipf_bias, gate=cfg.gate,
                     expert_bias=cfg.expert_bias,
                     mha=(dict(seq_len=cfg.seq_len, head_dim=cfg.head_dim, causal=cfg.causal)
                          if cfg.mha else None), device=dev)
    for name in ("x", "w_gate", "w1", "w3", "w2", "dy") + (("mha_in", "w_qkv", "w_o")
                                                           if cfg.mha else ()):
        if inp[name] is not None:
            getattr(layer, name).copy_(to_torch(inp[name], dev))
    for name in ("b1", "b3", "b2"):  # the experts' biases (fp32)
        if inp.get(name) is not None:
            getattr(layer, name).copy_(torch.from_numpy(inp[name]).to(dev))
    if cfg.zipf_bias:
        layer.bias.copy_(torch.from_numpy(inp["bias"]).to(dev))
    bufs = layer.bufs()
    # the layer runs on streams of its own (work on the legacy default stream
    # synchronises with every other stream)
    sc = torch.cuda.Stream()
    sm = sc if a.one_stream else torch.cuda.Stream()

    def step():
        layer.forward(sc, sm, bufs=bufs)
        layer.backward(sc, sm, bufs=bufs)

    for _ in range(a.warmup):
        step()
    torch.cuda.synchronize()

    # timed region: K steps, an event on the compute stream after every step
    # for the step time distribution
    step_ev = [torch.cuda.Event(enable_timing=True) for _ in range(a.steps + 1)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    step_ev[0].record(sc)
    for i in range(a.steps):
        step()
        step_ev[i + 1].record(sc)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    step_ms = sorted(step_ev[i].elapsed_time(step_ev[i + 1]) for i in range(a.steps))
    q = lambda f: float(np.percentile(step_ms, f))
    elapsed = t1 - t0

    # the same K steps again with every grouped-GEMM launch bracketed by HIP
    # events on its stream, for the per-launch durations (a timestamped event
    # around every launch adds ~2 us of idle per event to the step, so this
    # pass is kept out of the throughput)
    # (per step: ffn1, ffn2, dgrad1, dgrad2 per chunk; wgrad1, wgrad2 once)
    gemm_per_step = 4 * R + 2
    ev = EventArray(gemm_per_step * a.steps)
    L.flowmoe_trace_start(ev.ev, ev.kinds, ev.pairs, L.kind_mask(L.K_GEMM))
    torch.cuda.synchronize()
    t2 = time.perf_counter()
    for i in range(a.steps):
        step()
    torch.cuda.synchronize()
    t3 = time.perf_counter()
    n = L.flowmoe_trace_stop()
    gemm_ms = [ev.elapsed_ms(i) for i in range(n)]
    gemm_kinds = [L.K_NAMES[ev.kinds[i]] for i in range(n)]
    ev.close()
    # (work on the legacy default stream slows the layer's next ~20 steps:
    # this reduction waits until the timed passes are done)
    kept = int(layer.counts.sum().item())

    # untimed: one traced step over every kernel, for the per-kernel breakdown
    all_ev = EventArray(256)
    L.flowmoe_trace_start(all_ev.ev, all_ev.kinds, all_ev.pairs, 0xFFFFFFFF)
    step()
    torch.cuda.synchronize()
    m = L.flowmoe_trace_stop()
    per_kernel = {}
    for i in range(m):
        nm = L.K_NAMES[all_ev.kinds[i]]
        per_kernel.setdefault(nm, []).append(all_ev.elapsed_ms(i) * 1e3)
    all_ev.close()
    breakdown = {k: round(float(sum(v)), 2) for k, v in per_kernel.items()}  # us per step
    sched = schedule_overlap(layer, R, sc, sm, torch, cfg.mha)

    # the attention of AT_r: its kernels' durations over the K steps (HIP
    # events around each launch, a pass of its own) against their
    # algorithmic FLOPs
    attention = None
    if cfg.mha:
        akinds = ("attn_fwd", "attn_bwd_dq", "attn_bwd_dkdv", "attn_qkv", "attn_out",
                  "attn_dgrad", "attn_wgrad")
        aev = EventArray((7 * R + 2) * a.steps)
        L.flowmoe_trace_start(aev.ev, aev.kinds, aev.pairs, L.kind_mask(akinds))
        for i in range(a.steps):
            step()
        torch.cuda.synchronize()
        na = L.flowmoe_trace_stop()
        per = {}
        for i in range(na):
            per.setdefault(L.K_NAMES[aev.kinds[i]], []).append(aev.elapsed_ms(i))
        aev.close()
        af = attention_flops(cfg, R)
        ms = lambda *ks: sum(sum(per.get(k_, [])) for k_ in ks) / a.steps  # ms per step
        def rate(flops, t_ms):
            tf = flops / (t_ms * 1e-3) / 1e12 if t_ms > 0 else 0.0
            return {"ms_per_step": round(t_ms, 4), "TFLOPs": round(tf, 1),
                    "frac": round(tf / PEAK_BF16_TFLOPS, 4)}
        attention = {
            "shape": (f"{cfg.T // cfg.seq_len} sequences x {cfg.seq_len} tokens, {cfg.heads} "
                      f"heads of {cfg.head_dim}, {'causal' if cfg.causal else 'bidirectional'}"),
            "flops_per_step": af,
            "core_fwd": rate(af["core_fwd"], ms("attn_fwd")),
            "core_bwd": rate(af["core_bwd"], ms("attn_bwd_dq", "attn_bwd_dkdv")),
            "core_bwd_dq_ms": round(ms("attn_bwd_dq"), 4),
            "core_bwd_dkdv_ms": round(ms("attn_bwd_dkdv"), 4),
            "projections": rate(af["proj_fwd"] + af["proj_dgrad"] + af["proj_wgrad"],
                                ms("attn_qkv", "attn_out", "attn_dgrad", "attn_wgrad")),
            "launch_timing": "HIP events around every attention launch of a separate pass",
        }

    ms_per_step = elapsed / a.steps * 1e3
    tokens_per_s = cfg.T * a.steps / elapsed
    # algorithmic FLOPs of the traced launches: each row-mode launch covers
    # one chunk (its kept rows), each weight-gradient launch all R chunks;
    # chunks are enqueued once per step in a fixed order, so the launches of
    # one step come in the same order every step
    chunk_kept = [int(v) for v in layer.counts.sum(dim=1).tolist()]
    assert n == gemm_per_step * a.steps, (n, gemm_per_step, a.steps)
    tot_flops = 0.0
    for s0 in range(0, n, gemm_per_step):
        seen = {}
        for kd in gemm_kinds[s0:s0 + gemm_per_step]:
            if kd.startswith("wgrad"):
                tot_flops += gemm_flops(cfg, kd, kept)
            else:
                i = seen.get(kd, 0)
                seen[kd] = i + 1
                # forward kinds run chunks 0..R-1, backward kinds R-1..0
                r = i if kd in ("ffn1", "ffn2") else R - 1 - i
                tot_flops += gemm_flops(cfg, kd, chunk_kept[r])
    step_flops = gemm_flops_per_step(cfg, kept)
    assert abs(tot_flops - step_flops * a.steps) <= 1e-6 * step_flops * a.steps, (tot_flops, step_flops)
    fl = tot_flops / max(1, n)
    tot_s = sum(gemm_ms) / 1e3
    avg_launch_ms = sum(gemm_ms) / max(1, len(gemm_ms))
    achieved_tflops = tot_flops / tot_s / 1e12 if tot_s > 0 else 0.0

    mem = None
    if not a.no_memory_bound:
        flush = torch.ones(64 << 20, dtype=torch.int64, device=dev)  # 512 MiB
        mem = memory_bound(L, layer, cfg, torch, flush=flush)
        del flush

    if a.copy_probe > 0:
        n = a.copy_probe * 2**20 // 4
        src = torch.ones(n, device=dev, dtype=torch.float32)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    # HBM traffic of the grouped GEMM per launch, from the PMC passes kept
    # under profiles/ for this workload, if they were taken on this kernel source
    traffic, traffic_note = None, "no PMC summary for this workload"
    tpath = os.path.join(ROOT, "profiles", f"gemm_traffic_{cfg.name}.json")
    if os.path.exists(tpath):
        from paper_2510_00207_amd.profsum import gemm_source_hash
        tj = json.load(open(tpath))
        if tj.get("gemm_source_sha256") == gemm_source_hash():
            traffic = round(tj["gemm_bytes_per_launch"])
            traffic_note = (f"HBM bytes per launch (FETCH_SIZE x{tj['fetch_scale']} + WRITE_SIZE "
                            f"x{tj['write_scale']}, scaled by a {tj['probe_mib']} MiB copy probe)")
        else:
            traffic_note = "kernel changed since the PMC summary was taken"

    cpu = None
    if not a.no_cpu_baseline and not cfg.mha:  # (the headline line is the MoE layer's)
        import oracle
        from threadpoolctl import threadpool_info
        # a bounded sample of the same workload: the first Ts tokens, R
        # chunks of Ts / R, the same weights and capacity factor (whole steps
        # when they are cheap); weights widened to fp64 before the clock starts
        Ts = oracle_sample_tokens(cfg, R)
        i64 = {k: (None if v is None else (v.astype(np.float64) if k == "bias" else
                                           widen_f64(v[:Ts] if k in ("x", "dy") else v)))
               for k, v in inp.items()}
        del inp
        reps, c0 = 0, time.perf_counter()
        while True:
            oracle.layer_fwd_bwd(i64, k=cfg.k, f=cfg.f, act=cfg.act, R=R, layout=a.layout,
                                 gate=cfg.gate)
            reps += 1
            if time.perf_counter() - c0 >= 10.0 or reps >= 20:
                break
        c1 = time.perf_counter()
        threads = max([p.get("num_threads", 1) for p in threadpool_info()
                       if p.get("user_api") == "blas"] or [1])
        what = (f"{reps} full fwd+bwd step(s) of the {cfg.name} workload ({cfg.T} tokens each)"
                if Ts == cfg.T else
                f"{reps} fwd+bwd step(s) of the first {Ts} of the {cfg.name} workload's {cfg.T} "
                f"tokens ({R} chunk(s), capacity from f = {cfg.f} at that size, all {cfg.E} "
                f"experts' full weights)")
        cpu = {"value": round(Ts * reps / (c1 - c0), 2), "unit": "tokens/s", "cores": threads,
               "kind": "oracle", "sample": f"{what}, numpy fp64, {c1 - c0:.1f} s"}

    # the library's schedule: one chunk runs its forward on one stream, and its
    # backward on two only for layers whose expert GEMMs span many rounds
    if a.one_stream:
        streams = "1 stream"
    elif R > 1:
        streams = "2 streams"
    elif float(layer.rows) * cfg.M * cfg.H >= 2.5e11:
        streams = "1 stream forward, 2 backward"
    else:
        streams = "1 stream"
    out = {
        "metric": "MoE-layer fwd+bwd tokens/s on 1 MI355X; grouped-GEMM MFMA util %",
        "value": round(tokens_per_s, 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": a.steps,
        "warmup": a.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg.dtype,
        "data": "synthetic",
        "config": {
            "workload": (f"{cfg.name} MoE layer: T={cfg.T} M={cfg.M} H={cfg.H} E={cfg.E} "
                         f"top-{cfg.k} f={cfg.f} {cfg.act} {cfg.dtype}, R={R}, {a.layout}, "
                         f"{streams}"
                         f"{', full-softmax gate' if cfg.gate == 'full' else ''}"
                         f"{', biased experts' if cfg.expert_bias else ''}"
                         f"{'; AT_r with attention: ' + attention['shape'] if attention else ''}"),
            "T": cfg.T, "M": cfg.M, "H": cfg.H, "E": cfg.E, "k": cfg.k, "f": cfg.f,
            "C": layer.C, "R": R, "act": cfg.act, "layout": a.layout, "gate": cfg.gate, "tiles": a.tiles,
            "tile_order": a.tile_order,
            "expert_bias": cfg.expert_bias,
            "kept_rows": kept,
        },
        "roofline": {
            "kernel": f"grouped GEMM (gemm_dma_kernel, all {gemm_per_step} launches of a step)",
            "bound": "mfma",
            "achieved": round(achieved_tflops, 2),
            "peak": PEAK_BF16_TFLOPS,
            "unit": "TFLOP/s",
            "frac": round(achieved_tflops / PEAK_BF16_TFLOPS, 4),
            "traffic": traffic,
            "traffic_note": traffic_note,
            "flops_per_launch": fl,
            "flops_per_step": step_flops,
            "avg_launch_us": round(avg_launch_ms * 1e3, 2),
            "launches": len(gemm_ms),
            "launch_timing": (f"HIP events around every GEMM launch of a second pass of the "
                              f"{a.steps} steps ({(t3 - t2) / a.steps * 1e3:.4f} ms per step "
                              "with the events)"),
        },
        "gemm_mfma_util_pct": round(100 * achieved_tflops / PEAK_BF16_TFLOPS, 2),
        "step_ms_median": round(q(50), 4),
        "step_ms_iqr": [round(q(25), 4), round(q(75), 4)],
        "memory_bound": mem,
        "kernel_us_per_step": breakdown,
        "schedule": sched,
        "attention": attention,
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
