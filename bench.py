#!/usr/bin/env python3
"""Benchmark of one draft-and-verify iteration on one MI355X.

Workload: the 7B-shaped bf16 target (32 layers, d 4096, 32 heads x 128, SwiGLU
11008, vocab 32000) with a 4-layer draft (its first layers + shared embedding,
final norm and LM head), batch 1, resident context of 2048 positions,
gamma = 4, temperature 1.0.  A step is the whole iteration: gamma draft steps,
the verify pass, accept / resample, and the KV commit of both caches; every
step starts from the same context (the cache state is restored on the device
before each step), so all steps do identical work.

Reported value: verify-step tokens/s = batch*(gamma+1) / t_verify, where
t_verify covers specdec_verify + specdec_accept inside each timed step.
Weights and contexts are synthetic (seeded N(0, 0.02^2) weights drawn on the
device, N(0, (0.02 sqrt d)^2) K/V); the paper's trained models and datasets
are not used.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBPS = 8000.0
METRIC = "verify-step tokens/s (7B-shape, gamma=4, bs1); achieved HBM GB/s vs peak"


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--gamma", type=int, default=4)
    ap.add_argument("--ctx", type=int, default=2048)
    ap.add_argument("--batch", type=int, default=1)
    ap.add_argument("--temperature", type=float, default=1.0)
    ap.add_argument("--draft-layers", type=int, default=4)
    ap.add_argument("--no-graph", action="store_true", help="launch eagerly instead of replaying HIP graphs")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--profile-steps", type=int, default=5)
    ap.add_argument("--weights", choices=("bf16", "int4"), default="bf16",
                    help="layer weight format of the 7B verify line: bf16 (the headline), or INT4 codes with bf16 "
                         "scales per row and group of 128 columns (the paper's model precision)")
    ap.add_argument("--prefill", action="store_true",
                    help="prompt prefill on the 7B-shaped target: a 2048-token prompt in chunks of 64..512 rows")
    ap.add_argument("--config", type=int, default=3, choices=(1, 2, 3, 4, 5),
                    help="3 (default): the 7B gamma=4 bs1 headline line; 1: tiny float32; 2: 1.1B-shaped bf16; "
                         "4: draft switching (2/4/8-layer drafts, resident / reload / cache policy); "
                         "5: 7B-shaped, 16 sequences with contexts U[1024, 8192], gamma 6, T 0.8")
    ap.add_argument("--reload", action="store_true",
                    help="instead of the verify line, measure draft reloads (2/4/8-layer drafts) from pinned host "
                         "memory into a resident slot on a side stream, alone and under concurrent verify steps")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="also run one 1 GiB device-to-device copy (reference for the HBM byte counters)")
    ap.add_argument("--ceiling", action="store_true",
                    help="instead of the verify line, measure the streaming-read ceiling (64 MiB .. 4 GiB, cold)")
    ap.add_argument("--kernels-only", action="store_true",
                    help="only the 7B verify's kernels, each re-launched 20 times layer after layer, plus one 1 GiB "
                         "streaming read and one 1 GiB copy (the launches a counter profile of the kernels reads)")
    return ap.parse_args()


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


# ---------------------------------------------------------------- synthetic model on the device
def device_weights(shape, seed=0, weight_format="bf16"):
    """Seeded N(0, 0.02^2) bf16 weights drawn on the device (RMSNorm gains 1.0);
    weight_format "int4" packs the layer matrices as INT4 (quantized on the device)."""
    import torch
    from paper_2608_10362_amd import binding
    gen = torch.Generator(device="cuda")
    idx = [0]

    def mat(*shp):
        gen.manual_seed(seed * 1000003 + idx[0])
        idx[0] += 1
        t = torch.empty(shp, dtype=torch.float32, device="cuda").normal_(0.0, 0.02, generator=gen)
        return t.to(torch.bfloat16)

    def gain(n):
        idx[0] += 1
        return torch.ones(n, dtype=torch.bfloat16, device="cuda")

    d, f = shape.d_model, shape.ffn_dim
    w = {"embed": mat(shape.vocab, d), "layers": []}
    for _ in range(shape.n_layers):
        w["layers"].append({"attn_norm": gain(d), "wq": mat(shape.q_dim, d), "wk": mat(shape.kv_dim, d),
                            "wv": mat(shape.kv_dim, d), "wo": mat(d, shape.q_dim), "ffn_norm": gain(d),
                            "w_gate": mat(f, d), "w_up": mat(f, d), "w_down": mat(d, f)})
    w["final_norm"] = gain(d)
    w["lm_head"] = mat(shape.vocab, d)
    return binding.DeviceWeights(shape, w, weight_format=weight_format)


def install_context(kv, n_layers, shape, lengths, seed=5):
    import torch
    gen = torch.Generator(device="cuda")
    sigma = 0.02 * shape.d_model ** 0.5
    for l in range(n_layers):
        for b, L in enumerate(lengths):
            gen.manual_seed(seed * 7919 + l * 131 + b)
            k = (torch.randn((L, shape.n_kv_heads, shape.head_dim), generator=gen, device="cuda") * sigma)
            v = (torch.randn((L, shape.n_kv_heads, shape.head_dim), generator=gen, device="cuda") * sigma)
            kv.write_context(l, b, 0, k.to(torch.bfloat16), v.to(torch.bfloat16))


# ---------------------------------------------------------------- algorithmic bytes
def layer_weight_bytes(weights="bf16"):
    """Bytes per layer-matrix weight: bf16, or INT4 codes plus one bf16 scale per 128."""
    return 2.0 if weights == "bf16" else 0.5 + 2.0 / 128


def kernel_bytes(shape, ctx_read, weights="bf16"):
    """Algorithmic HBM bytes per launch of each kernel kind (weights streamed once,
    KV read for the keys a launch attends to); activations (a few hundred KB) left out."""
    d, f, V = shape.d_model, shape.ffn_dim, shape.vocab
    e = 2
    w = layer_weight_bytes(weights)
    return {
        "qkv": int((shape.q_dim + 2 * shape.kv_dim) * d * w) + d * e,
        "o_proj": int(d * shape.q_dim * w),
        "gate_up": int(2 * f * d * w) + d * e,
        "down": int(d * f * w),
        "lm_head": (V * d + d) * e,
        "attention": ctx_read * shape.n_kv_heads * shape.head_dim * 2 * e,
    }


def verify_step_bytes(shape, ctx, gamma, batch, weights="bf16"):
    """Bytes one verify step must move: every weight once, the committed KV, the new KV."""
    L, d, f, V = shape.n_layers, shape.d_model, shape.ffn_dim, shape.vocab
    e = 2
    per_layer = int(((shape.q_dim + 2 * shape.kv_dim) * d + d * shape.q_dim + 3 * f * d) * layer_weight_bytes(weights)) \
        + 2 * d * e
    weights = L * per_layer + (V * d + d) * e + batch * (gamma + 1) * d * e
    kv_row = shape.n_kv_heads * shape.head_dim * 2 * e * L
    return weights + batch * ctx * kv_row + batch * (gamma + 1) * kv_row


def measured_traffic(kernel: str):
    """HBM bytes per launch of a verify GEMM from the committed rocprofv3 counter summary
    (profiles/verify_7b_kernels_hbm_traffic.md), or None if absent or taken on other kernel source."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "verify_7b_kernels_hbm_traffic.md")
    if not os.path.exists(path):
        return None
    fields = {}
    for line in open(path):
        if ":" in line and not line.startswith(("|", "#", "`", "-")):
            k, v = line.split(":", 1)
            fields[k.strip()] = v.strip()
    src = os.path.join(ROOT, "paper_2608_10362_amd", "csrc", "gemm.hip")
    if not os.path.exists(src):
        return None
    sha = hashlib.sha256(open(src, "rb").read()).hexdigest()
    if fields.get("kernel_source_sha256") != sha or f"traffic_{kernel}" not in fields:
        return None
    return int(float(fields[f"traffic_{kernel}"]))


# ---------------------------------------------------------------- streaming-read ceiling
def read_ceiling(sizes_mib=(64, 256, 1024, 4096), buf_gib=8, reps=5):
    """Read rate of the library's streaming-read probe (specdec_stream_read: the
    weight stream's access pattern) over cold regions of an 8 GiB buffer: each
    timed launch reads a region the launches just before it did not touch (the
    last-level cache holds 256 MB).  Median of `reps` launches after one warm-up,
    HIP events on the launch stream."""
    import torch
    from paper_2608_10362_amd import binding
    buf = torch.empty(buf_gib << 30, dtype=torch.uint8, device="cuda")
    sink = torch.zeros(1, dtype=torch.int32, device="cuda")
    s = torch.cuda.current_stream()
    out = {}
    for mib in sizes_mib:
        n = mib << 20
        regions = (buf_gib << 30) // n
        times = []
        for r in range(reps + 1):
            off = ((r * 2) % regions) * n  # (every other region: no neighbour left in the cache)
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(s)
            binding.specdec_stream_read(buf[off:off + n], sink, stream=s)
            e1.record(s)
            e1.synchronize()
            if r > 0:
                times.append(e0.elapsed_time(e1) * 1e-3)
        t = float(np.median(times))
        out[f"{mib}MiB"] = {"bytes": n, "us": round(t * 1e6, 2), "GBps": round(n / t / 1e9, 1)}
    del buf
    torch.cuda.empty_cache()
    return out


# ---------------------------------------------------------------- CPU oracle baseline
def cpu_baseline(shape, ctx, gamma):
    """The oracle's verify pass on the host: time 2 and 6 layers (+ final norm and
    LM head) of the 7B shape at the same context, five runs each (about 10 s of
    oracle time), and extrapolate the per-layer time to all layers."""
    import numpy as np
    from threadpoolctl import threadpool_info

    from oracle import model as om
    from paper_2608_10362_amd import synth

    L0, L1, runs = 2, 6, 5
    W = synth.make_weights(shape, n_layers=L1, threads=min(16, os.cpu_count() or 1))
    ctxkv = synth.make_kv_context(shape, L1, [ctx], threads=min(16, os.cpu_count() or 1))
    toks = [int(t) for t in synth.make_prompt(gamma + 1, shape.vocab)[0]]
    times = {}
    for L in (L0, L1):
        best = []
        for _ in range(runs):
            c = om.KVCache(shape, L, ctx + gamma + 1)
            for l in range(L):
                c.load(l, ctxkv[l][0]["k"], ctxkv[l][0]["v"])
            c.length = ctx
            m = om.Model(shape, W, n_layers=L)
            t0 = time.perf_counter()
            m.forward_block(toks, ctx, c)
            best.append(time.perf_counter() - t0)
        times[L] = float(np.median(best))
    t_layer = max((times[L1] - times[L0]) / (L1 - L0), 1e-9)
    t_rest = max(times[L0] - L0 * t_layer, 0.0)
    t_full = t_rest + shape.n_layers * t_layer
    threads = [i.get("num_threads", 1) for i in threadpool_info() if i.get("user_api") == "blas"]
    return {"value": (gamma + 1) / t_full, "unit": "tokens/s", "cores": int(max(threads) if threads else 1),
            "kind": "oracle",
            "sample": (f"float64 numpy oracle verify pass (gamma={gamma}, ctx {ctx}) over {L0} and {L1} layers of the "
                       f"7B shape + LM head, median of {runs} runs each ({times[L0]:.2f} s, {times[L1]:.2f} s); "
                       f"per-layer time x {shape.n_layers} layers -> {t_full:.1f} s per verify step")}


# ---------------------------------------------------------------- draft reload
def reload_bench(dw, graphs, verify_part, args):
    """H2D reloads of 2/4/8-layer draft layers into one resident slot (the LM
    head stays in the slot), each timed with events on the copy stream; then
    the verify step replayed on the main stream while an 8-layer reload runs
    on the side stream, against the verify step alone."""
    import numpy as np
    import torch

    from paper_2608_10362_amd import binding
    slot = binding.DraftSlot(dw, max_layers=8)
    copy = torch.cuda.Stream()
    torch.cuda.synchronize()
    log(f"draft slot {slot.nbytes / 1e9:.2f} GB, pinned host image {slot.host.numel() / 1e9:.2f} GB")

    def timed_load(k):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(copy)
        nb = slot.load_async(k, copy)
        e1.record(copy)
        return nb, e0, e1

    loads = {}
    for k in (2, 4, 8):
        ms = []
        for _ in range(3):
            nb, e0, e1 = timed_load(k)
            e1.synchronize()
            ms.append(e0.elapsed_time(e1))
        med = float(np.median(ms))
        loads[str(k)] = {"bytes": nb, "ms": round(med, 3), "GBps": round(nb / (med * 1e-3) / 1e9, 2)}
    nb, e0, e1 = timed_load(8)
    issued_not_done = not slot.event.query()  # the load is asynchronous: the host was not blocked
    e1.synchronize()

    def replay_verify():
        if graphs:
            graphs[1].replay()
        else:
            verify_part(0)

    for _ in range(5):
        replay_verify()
    torch.cuda.synchronize()
    n = 10
    a0, a1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a0.record()
    for _ in range(n):
        replay_verify()
    a1.record()
    a1.synchronize()
    alone = a0.elapsed_time(a1) / n
    # as many verify steps as fit inside one 8-layer reload
    n_ov = max(1, int(loads["8"]["ms"] / alone) - 2)
    torch.cuda.synchronize()
    nb, e0, e1 = timed_load(8)
    b0, b1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    b0.record()
    for _ in range(n_ov):
        replay_verify()
    b1.record()
    torch.cuda.synchronize()
    during = b0.elapsed_time(b1) / n_ov
    copy_ms = e0.elapsed_time(e1)
    return {
        "metric": "draft reload into a resident slot (H2D, side stream)",
        "unit": "ms",
        "higher_is_better": False,
        "data": "synthetic",
        "dtype": "bf16",
        "config": {"workload": "7B-shaped target; 2/4/8-layer draft layers copied from pinned host memory into one "
                               "HBM slot that keeps the shared LM head", "slot_bytes": slot.nbytes},
        "reload": loads,
        "load_returned_before_completion": bool(issued_not_done),
        "verify_ms_alone": round(alone, 4),
        "verify_ms_during_8_layer_reload": round(during, 4),
        "verify_steps_overlapped": n_ov,
        "reload_ms_under_verify": round(copy_ms, 3),
        "hip_graph": bool(graphs),
    }


# ---------------------------------------------------------------- shared step timing
def capture_graphs(sd, draft_part, verify_part, commit_part, no_graph):
    """Capture draft / verify+accept / commit as three HIP graphs; every replay is
    checked bit for bit against an eager step (three replays, eager work in
    between).  Returns None (eager launches) if capture is off or fails."""
    import torch
    draft_part(0); verify_part(0); commit_part()
    torch.cuda.synchronize()
    ref = (sd.d.clone(), sd.logits.clone(), sd.n_acc.clone(), sd.next.clone())
    if no_graph:
        return None
    try:
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            draft_part(0); verify_part(0); commit_part()
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        gd, gv, gc = torch.cuda.CUDAGraph(), torch.cuda.CUDAGraph(), torch.cuda.CUDAGraph()
        with torch.cuda.graph(gd):
            draft_part(0)
        with torch.cuda.graph(gv):
            verify_part(0)
        with torch.cuda.graph(gc):
            commit_part()
        for r in range(3):
            gd.replay(); gv.replay(); gc.replay()
            torch.cuda.synchronize()
            same = (torch.equal(sd.d, ref[0]) and torch.equal(sd.logits, ref[1]) and
                    torch.equal(sd.n_acc, ref[2]) and torch.equal(sd.next, ref[3]))
            if not same:
                raise RuntimeError(f"graph replay {r} differs from the eager step")
            draft_part(0); verify_part(0); commit_part()
            torch.cuda.synchronize()
        return (gd, gv, gc)
    except Exception as e:
        log(f"graph capture disabled: {e}")
        return None


def time_steps(graphs, draft_part, verify_part, commit_part, steps, warmup):
    """Time `steps` steps after `warmup`: the verify (+ accept) time from events
    around the verify graph, the step time from events around the loop."""
    import torch

    def run_step(i, ev=None):
        if graphs:
            graphs[0].replay()
            if ev: ev[0].record()
            graphs[1].replay()
            if ev: ev[1].record()
            graphs[2].replay()
        else:
            draft_part(i)
            if ev: ev[0].record()
            verify_part(i)
            if ev: ev[1].record()
            commit_part()

    for i in range(warmup):
        run_step(i)
    torch.cuda.synchronize()
    evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
    start, end = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    start.record()
    for i in range(steps):
        run_step(warmup + i, evs[i])
    end.record()
    torch.cuda.synchronize()
    verify = [a.elapsed_time(b) for a, b in evs]
    return {"verify_ms": sum(verify) / steps, "verify_ms_p10": float(np.percentile(verify, 10)),
            "verify_ms_p50": float(np.percentile(verify, 50)), "verify_ms_p90": float(np.percentile(verify, 90)),
            "step_ms": start.elapsed_time(end) / steps}


def verify_bytes_ragged(shape, lengths, gamma):
    """verify_step_bytes for per-sequence contexts."""
    L, d, f, V = shape.n_layers, shape.d_model, shape.ffn_dim, shape.vocab
    e = 2 if shape.dtype == "bf16" else 4
    B = len(lengths)
    per_layer = ((shape.q_dim + 2 * shape.kv_dim) * d + d * shape.q_dim + 3 * f * d + 2 * d) * e
    weights = L * per_layer + (V * d + d) * e + B * (gamma + 1) * d * e
    kv_row = shape.n_kv_heads * shape.head_dim * 2 * e * L
    return weights + int(sum(lengths)) * kv_row + B * (gamma + 1) * kv_row


CONFIGS = {
    1: dict(metric_name="tiny float32 model", desc="tiny float32 (L=2, d=128, 4x32 MHA, F=512, V=512), 1-layer draft, 64-token prompt",
            shape="TINY", batch=1, gamma=4, prompt=64, temperature=1.0, draft_layers=1, generate=32),
    2: dict(metric_name="1.1B-shaped, batch 1", desc="1.1B-shaped bf16 (L=22, d=2048, 32q/4kv x 64, F=5632, V=32000), 4-layer draft, "
                 "512-token prompt", shape="LLAMA_1B", batch=1, gamma=4, prompt=512, temperature=1.0,
            draft_layers=4, generate=256),
    5: dict(metric_name="7B-shaped, 16 long-context sequences", desc="7B-shaped bf16, 16 sequences with resident contexts U[1024, 8192] (seed 4), 4-layer draft",
            shape="LLAMA_7B", batch=16, gamma=6, lengths=(1024, 8192), temperature=0.8, draft_layers=4),
}


def run_config(args):
    """Configurations other than the headline one, measured the same way: every
    step from the same state (restored on the device), graph replays, HIP events."""
    import torch

    from paper_2608_10362_amd import binding, synth
    cfg = CONFIGS[args.config]
    shape = getattr(synth, cfg["shape"])
    B, g, T, k = cfg["batch"], cfg["gamma"], cfg["temperature"], cfg["draft_layers"]
    t0 = time.time()
    if shape.dtype == "f32":
        dw = binding.DeviceWeights(shape, synth.make_weights(shape))
    else:
        dw = device_weights(shape)
    if "prompt" in cfg:
        n0 = cfg["prompt"]
        lengths = np.full(B, n0 - 1, np.int64)
        need = n0 + cfg["generate"] + 2 * g + 2
    else:
        lengths = synth.make_ragged_lengths(B, *cfg["lengths"]).astype(np.int64)
        need = int(lengths.max()) + g + 2
    cap = (need + 63) // 64 * 64
    rows = max(B * (g + 1), 2 * B, 64)
    target = binding.Model(dw, shape.n_layers, max_rows=rows, max_ctx=cap)
    draft = binding.Model(dw, k, max_rows=rows, max_ctx=cap)
    kv_t, kv_d = binding.KVCache(target, B, cap), binding.KVCache(draft, B, cap)
    if "prompt" in cfg:
        tok = torch.from_numpy(synth.make_prompt(cfg["prompt"], shape.vocab, batch=B).astype(np.int32)).cuda()
        binding.specdec_prefill(target, kv_t, tok)
        binding.specdec_prefill(draft, kv_d, tok)
    else:
        install_context(kv_t, shape.n_layers, shape, [int(x) for x in lengths])
        install_context(kv_d, k, shape, [int(x) for x in lengths])
        pend = synth.make_prompt(1, shape.vocab, batch=B)[:, 0]
        st = (lengths.astype(np.int32), np.stack([np.zeros(B, np.int32), pend], 1), np.ones(B, np.int32))
        kv_t.set_state(*st)
        kv_d.set_state(*st)
    torch.cuda.synchronize()
    saved = (kv_t.state.clone(), kv_d.state.clone(), kv_t.kv.len_upper, kv_d.kv.len_upper)
    sd = binding.SpecDecoder(target, draft, kv_t, kv_d, g, T, seed=synth.SEED_SAMPLING)
    log(f"config {args.config} set-up {time.time() - t0:.1f} s")

    def restore():
        kv_t.state.copy_(saved[0]); kv_d.state.copy_(saved[1])
        kv_t.kv.len_upper, kv_d.kv.len_upper = saved[2], saved[3]

    def draft_part(i):
        restore()
        sd.draft_phase(i)

    verify_part = lambda i: sd.verify_phase(i)  # noqa: E731
    graphs = capture_graphs(sd, draft_part, verify_part, sd.commit_phase, args.no_graph)
    tm = time_steps(graphs, draft_part, verify_part, sd.commit_phase, args.steps, args.warmup)
    status = min(int(sd.status.item()), kv_t.read_state()["status"], kv_d.read_state()["status"])
    acc = []
    for i in range(8):
        draft_part(1000 + i); sd.verify_phase(1000 + i); sd.commit_phase()
        acc.append(sd.n_acc.clone())
    mean_A = float(torch.stack(acc).float().mean().item())
    vbytes = verify_bytes_ragged(shape, lengths, g)
    gbps = vbytes / (tm["verify_ms"] * 1e-3) / 1e9
    result = {
        "metric": f"verify-step tokens/s ({cfg['metric_name']})", "value": round(B * (g + 1) / (tm["verify_ms"] * 1e-3), 2),
        "unit": "tokens/s", "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(tm["step_ms"], 4), "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "bf16" if shape.dtype == "bf16" else "f32", "data": "synthetic",
        "config": {"workload": cfg["desc"], "gamma": g, "batch": B, "temperature": T, "draft_layers": k,
                   "context_lengths": [int(x) for x in lengths][:16], "hip_graph": bool(graphs)},
        "verify_ms": round(tm["verify_ms"], 4), "verify_ms_p10_p50_p90": [round(tm["verify_ms_p10"], 4),
                                                                         round(tm["verify_ms_p50"], 4),
                                                                         round(tm["verify_ms_p90"], 4)],
        "verify_bytes": vbytes, "verify_hbm_GBps": round(gbps, 1), "verify_hbm_frac": round(gbps / PEAK_HBM_GBPS, 4),
        "generated_tokens_per_s": round(B * (mean_A + 1) / (tm["step_ms"] * 1e-3), 2),
        "mean_accepted": round(mean_A, 3), "device_status": status,
    }
    print(json.dumps(result), flush=True)


# ---------------------------------------------------------------- draft switching
def run_switching(args):
    """Draft switching on the 7B-shaped target (Sec. 3.3-3.4 on one GPU): drafts
    of 2, 4 and 8 layers, context 1024, gamma 4, greedy, scheduling every N = 4
    iterations along a Markov schedule (stay 0.8, seed 3, starting at the
    4-layer draft), 128 generated tokens.  Modes: static (the 4-layer draft
    throughout), resident (every draft resident), reload (one slot, blocking
    reload on a switch), memspec (K = 2 slots, Alg. 2 prefetches overlapped with
    decoding, best resident draft, Alg. 3), mab (K = 2 slots, the MAB-Async
    baseline: UCB with c = 2.0 over observed utilities, reactive asynchronous
    loads, the active draft as the fallback).  Wall time covers the whole run,
    catch-up forwards and reloads included."""
    import torch

    from paper_2608_10362_amd import binding, synth
    from paper_2608_10362_amd.runtime import HostImage, SwitchingRunner, observed_utility, score_stream
    shape = synth.LLAMA_7B
    layers, g, ctx, N, K, n_iter, n_tok = [2, 4, 8], 4, 1024, 4, 2, 400, 128
    cap = (ctx + n_iter * (g + 1) + 2 * g + 63) // 64 * 64
    dw = device_weights(shape)
    image = HostImage(dw, max(layers))
    points = (n_iter + N - 1) // N
    schedule = synth.make_markov_schedule(points, 3, start=1, stay=0.8)
    scores = score_stream(schedule, 3)
    utility = observed_utility(schedule, 3)
    pend = int(synth.make_prompt(1, shape.vocab)[0, 0])
    out = {}
    ref_text = None
    for mode in ("static", "resident", "reload", "memspec", "mab"):
        target = binding.Model(dw, shape.n_layers, max_rows=g + 1, max_ctx=cap)
        kv_t = binding.KVCache(target, 1, cap)
        r = SwitchingRunner(dw, target, kv_t, layers, g, 0.0, synth.SEED_SAMPLING, cap,
                            "resident" if mode == "static" else mode, slots=K if mode in ("memspec", "mab") else 1,
                            image=image)
        install_context(kv_t, shape.n_layers, shape, [ctx])
        for d, k in enumerate(layers):
            install_context(r.kv[d], k, shape, [ctx])
        r.start_from_context(ctx, pend)
        sched = [1] * points if mode == "static" else list(schedule)
        st = r.run(n_iter, sched, scores, N, max_tokens=n_tok, utility=utility)
        text = r.text[ctx:]
        if ref_text is None:
            ref_text = text
        n_common = min(len(text), len(ref_text))
        same = text[:n_common] == ref_text[:n_common]
        out[mode] = {"wall_ms": round(st.wall_ms, 2), "iterations": st.iterations, "tokens": st.tokens,
                     "tokens_per_s": round(st.tokens / (st.wall_ms * 1e-3), 2), "switches": st.switches,
                     "reloads": st.reloads, "reload_GB": round(st.reload_bytes / 1e9, 3),
                     "blocked_ms": round(st.blocked_ms, 2), "catchup_tokens": st.catchup_tokens,
                     "matches_desired": round(float(np.mean([a == d for a, d in zip(st.active, st.desired)])), 3),
                     "fallback_fraction": round(st.fallback_fraction(), 3),
                     "desired_ms": round(st.desired_ms, 2), "fallback_ms": round(st.fallback_ms, 2),
                     "prediction_ms": round(st.prediction_ms, 3),
                     "time_breakdown": {k: round(v, 4) for k, v in st.time_breakdown().items()},
                     "text_agrees": bool(same)}
        log(f"{mode}: {out[mode]}")
        del r, target, kv_t
        torch.cuda.empty_cache()
    result = {
        "metric": "generated tokens/s under draft switching (7B target, 2/4/8-layer drafts)", "value": out["memspec"]["tokens_per_s"],
        "unit": "tokens/s", "n_gpus": 1, "higher_is_better": True, "data": "synthetic", "dtype": "bf16",
        "config": {"workload": "7B-shaped bf16 target, drafts of 2/4/8 layers, context 1024, gamma 4, greedy, "
                               "interval N=4, K=2, Markov schedule stay 0.8 (seed 3), 128 generated tokens",
                   "draft_layers": layers},
        "modes": out,
    }
    print(json.dumps(result), flush=True)


# ---------------------------------------------------------------- prefill (large-M path)
def run_prefill(args):
    """Prefill of a 2048-token prompt on the 7B-shaped bf16 target (32 layers),
    in chunks of 64, 128, 256 and 512 rows (the handle's max_rows): chunks of
    more than 64 rows run the wide GEMM in launches of up to 128 rows and the
    looping attention.  Eager launches timed with HIP events, best of 3 after a
    warm-up; the cache length is reset between runs."""
    import torch

    from paper_2608_10362_amd import binding, synth
    shape = synth.LLAMA_7B
    n = 2048
    dw = device_weights(shape)
    tok = torch.from_numpy(synth.make_prompt(n, shape.vocab)).cuda()
    d, f = shape.d_model, shape.ffn_dim
    # linear-layer flops per token (2 per multiply-add) and attention flops over the causal prefix
    lin = 2 * (shape.n_layers * (d * (shape.q_dim + 2 * shape.kv_dim) + shape.q_dim * d + 3 * d * f) + d * shape.vocab)
    attn = shape.n_layers * 2 * 2 * shape.q_dim * (n - 1) * n / 2
    flops = lin * (n - 1) + attn
    out = {}
    for rows in (64, 128, 256, 512):
        target = binding.Model(dw, shape.n_layers, max_rows=rows, max_ctx=n + 64)
        kv = binding.KVCache(target, 1, n + 64)
        times = []
        for rep_i in range(4):
            kv.set_state(np.zeros(1, np.int32), np.zeros((1, 2), np.int32), np.ones(1, np.int32))
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            torch.cuda.synchronize()
            e0.record()
            binding.specdec_prefill(target, kv, tok)
            e1.record()
            torch.cuda.synchronize()
            if rep_i:
                times.append(e0.elapsed_time(e1))
        st = kv.read_state()
        assert int(st["len"][0]) == n - 1 and int(st["status"]) == 0
        ms = min(times)
        out[rows] = {"ms": round(ms, 3), "tokens_per_s": round((n - 1) / (ms * 1e-3), 1),
                     "TFLOPs": round(flops / (ms * 1e-3) / 1e12, 1)}
        log(f"prefill rows {rows}: {out[rows]}")
        del target, kv
        torch.cuda.empty_cache()
    best = min(out, key=lambda r: out[r]["ms"])
    result = {
        "metric": "prefill tokens/s (7B-shape bf16, 2048-token prompt)", "value": out[best]["tokens_per_s"],
        "unit": "tokens/s", "n_gpus": 1, "higher_is_better": True, "data": "synthetic", "dtype": "bf16",
        "config": {"workload": "7B-shaped bf16 target (32 layers), one 2048-token prompt, chunked prefill",
                   "best_chunk_rows": best},
        "flops_per_prefill": flops,
        "roofline": {"bound": "mfma", "achieved": out[best]["TFLOPs"], "peak": 2500.0, "unit": "TFLOP/s",
                     "frac": round(out[best]["TFLOPs"] / 2500.0, 4), "traffic": None,
                     "note": "float32 activations take two bf16 products per weight (hi + lo split)"},
        "chunks": out,
    }
    print(json.dumps(result), flush=True)


# ---------------------------------------------------------------- main
def run_kernels_only(args, shape, B, g, ctx, cap):
    """The verify pass's kernels alone (no draft, no graphs): one verify, then
    each kernel kind re-launched 20 times by specdec_time_kernel (launch i runs
    layer i mod 32, cold weights), then one 1 GiB streaming read and one 1 GiB
    device copy.  Prints the per-kind average durations."""
    import torch
    from paper_2608_10362_amd import binding, synth
    dw = device_weights(shape)
    target = binding.Model(dw, shape.n_layers, max_rows=B * (g + 1), max_ctx=cap)
    kv_t = binding.KVCache(target, B, cap)
    install_context(kv_t, shape.n_layers, shape, [ctx] * B)
    pend = synth.make_prompt(1, shape.vocab, batch=B)[:, 0]
    kv_t.set_state(np.full(B, ctx, np.int32), np.stack([np.zeros(B, np.int32), pend], 1), np.ones(B, np.int32))
    drafts = torch.from_numpy(synth.make_prompt(g, shape.vocab, batch=B, seed=32)).cuda()
    logits = torch.empty((B, g + 1, shape.vocab), dtype=torch.float32, device="cuda")
    binding.specdec_verify(target, kv_t, g, drafts, g, logits)
    torch.cuda.synchronize()
    kb = kernel_bytes(shape, ctx + g + 1)
    out = {}
    for k in ("embed", "qkv", "attention", "o_proj", "gate_up", "down", "lm_head"):
        us = binding.specdec_time_kernel(target, k, reps=20)
        out[k] = {"avg_us": round(us, 3), "launches": 20, "bytes": kb.get(k)}
        log(f"{k}: {us:.2f} us")
    src = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
    sink = torch.zeros(1, dtype=torch.int32, device="cuda")
    binding.specdec_stream_read(src, sink)
    dst = torch.empty_like(src)
    dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"metric": "7B verify kernels, re-launched layer after layer", "kernels": out,
                      "config": {"workload": f"7B-shaped bf16 verify, gamma={g}, batch {B}, context {ctx}"}}),
          flush=True)


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU: the library has no multi-GPU path (asked for --gpus {args.gpus}).",
              file=sys.stderr)
        sys.exit(2)
    import torch

    from paper_2608_10362_amd import binding, synth

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    binding.lib()
    if args.prefill:
        run_prefill(args)
        return
    if args.ceiling:
        rc = read_ceiling()
        print(json.dumps({"metric": "streaming-read ceiling (specdec_stream_read, cold regions)",
                          "value": rc["1024MiB"]["GBps"], "unit": "GB/s", "n_gpus": 1, "peak_GBps": PEAK_HBM_GBPS,
                          "frac_of_peak": round(rc["1024MiB"]["GBps"] / PEAK_HBM_GBPS, 4), "sizes": rc}), flush=True)
        return
    if args.config == 4:
        run_switching(args)
        return
    if args.config != 3:
        run_config(args)
        return
    shape = synth.LLAMA_7B
    B, g, ctx, T = args.batch, args.gamma, args.ctx, args.temperature
    cap = ((ctx + g + 2 + 63) // 64) * 64
    if args.kernels_only:
        run_kernels_only(args, shape, B, g, ctx, cap)
        return
    t0 = time.time()
    dw = device_weights(shape, weight_format=args.weights)
    target = binding.Model(dw, shape.n_layers, max_rows=max(B * (g + 1), 2 * B), max_ctx=cap)
    draft = binding.Model(dw, args.draft_layers, max_rows=max(B * (g + 1), 2 * B), max_ctx=cap)
    kv_t = binding.KVCache(target, B, cap)
    kv_d = binding.KVCache(draft, B, cap)
    install_context(kv_t, shape.n_layers, shape, [ctx] * B)
    install_context(kv_d, args.draft_layers, shape, [ctx] * B)
    pend = synth.make_prompt(1, shape.vocab, batch=B)[:, 0]
    st = (np.full(B, ctx, np.int32), np.stack([np.zeros(B, np.int32), pend], 1), np.ones(B, np.int32))
    kv_t.set_state(*st)
    kv_d.set_state(*st)
    saved_t, saved_d = kv_t.state.clone(), kv_d.state.clone()
    sd = binding.SpecDecoder(target, draft, kv_t, kv_d, g, T, seed=synth.SEED_SAMPLING)
    torch.cuda.synchronize()
    log(f"set-up {time.time() - t0:.1f} s (packed weight image {dw.packed.numel() / 1e9:.2f} GB)")

    def restore():
        kv_t.state.copy_(saved_t)
        kv_d.state.copy_(saved_d)
        kv_t.kv.len_upper = ctx
        kv_d.kv.len_upper = ctx

    def draft_part(i):
        restore()
        sd.draft_phase(i)

    def verify_part(i):
        sd.verify_phase(i)

    def commit_part():
        sd.commit_phase()

    graphs = capture_graphs(sd, draft_part, verify_part, commit_part, args.no_graph)
    use_graph = graphs is not None
    if args.reload:
        print(json.dumps(reload_bench(dw, graphs, verify_part, args)), flush=True)
        return
    tm = time_steps(graphs, draft_part, verify_part, commit_part, args.steps, args.warmup)
    verify_ms, step_ms = tm["verify_ms"], tm["step_ms"]
    status = min(int(sd.status.item()), kv_t.read_state()["status"], kv_d.read_state()["status"])

    # mean accepted length over eager steps with distinct random draws (outside the timed region)
    acc = []
    for i in range(8):
        draft_part(1000 + i); verify_part(1000 + i); commit_part()
        acc.append(sd.n_acc.clone())
    mean_A = float(torch.stack(acc).float().mean().item())

    if args.copy_calibration:  # a plain copy of known size for scaling FETCH_SIZE / WRITE_SIZE
        src = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    # Whole-step profile: every launch bracketed by HIP events on the library's stream
    # (adds a few us per launch; used for the step breakdown only).
    binding.specdec_timing_enable(True)
    for i in range(args.profile_steps):
        draft_part(i); verify_part(i); commit_part()
    torch.cuda.synchronize()
    per = binding.specdec_timing_read()
    binding.specdec_timing_enable(False)
    step_profile = {k: {"ms_per_step": round(ms / args.profile_steps, 4),
                        "launches_per_step": n / args.profile_steps} for k, (ms, n) in per.items() if n}

    # Per-kernel durations of the verify pass: each kernel re-launched back to back
    # between HIP events on the library's stream, layer after layer (so every launch
    # streams weights and keys/values the launches before it did not touch).
    draft_part(0); verify_part(0)
    torch.cuda.synchronize()
    kb_verify = kernel_bytes(shape, ctx + g + 1, args.weights)
    # (bf16: RoPE and the KV append run in the QKV GEMM's epilogue, no rope_append launch)
    per_layer = {"embed": 1, "qkv": shape.n_layers, "attention": shape.n_layers,
                 "o_proj": shape.n_layers, "gate_up": shape.n_layers, "down": shape.n_layers, "lm_head": 1}
    kernels = {}
    for k, n in per_layer.items():
        us = binding.specdec_time_kernel(target, k, reps=20)
        entry = {"avg_us": round(us, 3), "launches_per_verify": n, "ms_per_verify": round(us * n / 1e3, 4)}
        if k in kb_verify:
            entry["bytes"] = kb_verify[k]
            entry["GBps"] = round(kb_verify[k] / (us * 1e-6) / 1e9, 1)
        kernels[k] = entry
    dom = max((k for k in kernels if k in kb_verify and k != "attention"), key=lambda k: kernels[k]["ms_per_verify"])
    dom_bytes = kb_verify[dom]
    achieved = dom_bytes / (kernels[dom]["avg_us"] * 1e-6) / 1e9
    vbytes = verify_step_bytes(shape, ctx, g, B, args.weights)
    verify_GBps = vbytes / (verify_ms * 1e-3) / 1e9
    ceiling = read_ceiling(sizes_mib=(1024,))["1024MiB"]
    int4 = args.weights == "int4"

    result = {
        "metric": METRIC if not int4 else "verify-step tokens/s (7B-shape, INT4 g128 layer weights, gamma=4, bs1)",
        "value": round(B * (g + 1) / (verify_ms * 1e-3), 2),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(step_ms, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"7B-shaped {'INT4-g128' if int4 else 'bf16'} target verify + "
                               f"{args.draft_layers}-layer draft, gamma={g}, batch {B}, context {ctx}, temperature {T}",
                   "gamma": g, "batch": B, "ctx": ctx, "temperature": T, "draft_layers": args.draft_layers,
                   "hip_graph": use_graph, "weights": args.weights},
        "roofline": {"bound": "hbm", "kernel": f"gemm {dom}", "achieved": round(achieved, 1),
                     "peak": PEAK_HBM_GBPS, "unit": "GB/s", "frac": round(achieved / PEAK_HBM_GBPS, 4),
                     "traffic": None if int4 else measured_traffic(dom), "bytes_per_launch": dom_bytes,
                     # the whole verify step (verify + accept) against the same peak
                     "step": {"achieved": round(verify_GBps, 1), "frac": round(verify_GBps / PEAK_HBM_GBPS, 4),
                              "bytes": vbytes, "ms": round(verify_ms, 4),
                              "frac_of_read_ceiling": round(verify_GBps / ceiling["GBps"], 4)},
                     # the same device's streaming-read rate for the weight stream's access pattern
                     "read_ceiling": {"GBps": ceiling["GBps"], "frac_of_peak": round(ceiling["GBps"] / PEAK_HBM_GBPS, 4),
                                      "bytes": ceiling["bytes"], "kernel": "specdec_stream_read"}},
        "verify_ms": round(verify_ms, 4),
        "verify_ms_p10_p50_p90": [round(tm["verify_ms_p10"], 4), round(tm["verify_ms_p50"], 4),
                                  round(tm["verify_ms_p90"], 4)],
        "verify_hbm_GBps": round(verify_GBps, 1),
        "verify_hbm_frac": round(verify_GBps / PEAK_HBM_GBPS, 4),
        "verify_frac_of_read_ceiling": round(verify_GBps / ceiling["GBps"], 4),
        "verify_bytes": vbytes,
        "generated_tokens_per_s": round(B * (mean_A + 1) / (step_ms * 1e-3), 2),
        "mean_accepted": round(mean_A, 3),
        "device_status": status,
        "kernels": kernels,
        "step_profile": step_profile,
    }
    if not args.no_cpu_baseline and not int4:
        log("timing the CPU oracle baseline")
        result["cpu_baseline"] = cpu_baseline(shape, ctx, g)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
