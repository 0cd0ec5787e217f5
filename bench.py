"""Benchmark: MoE decode tokens/s under a 6 GiB expert budget on one MI355X.

Default workload: 40 decode layers of a 128-expert top-8 MoE (hidden 2048,
expert intermediate 768, bf16 weights), all 48.3 GB of routed experts in pinned
host memory, 682 expert slots in HBM (6 GiB), LRU residency, Zipf(1.1)
routing with 70 % overlap between consecutive tokens, batch 1.  A step is one
token through all 40 layers (pre-norm, route, slot lookup and fills, expert FFN
with fused combine and residual).  Prints one JSON line.

--config 5: 48 layers of 256 int4 experts (group-128 scales) top-8 plus a shared
expert, 6 GiB budget (3923 slots): a 2048-token prompt chunk (grouped MFMA
GEMMs) from a cold cache, then 512 batch-1 decode steps; both are timed and
reported, the decode rate being `value`.
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

METRIC = "MoE decode tokens/sec at batch 1 under 6 GB expert budget; expert-FFN HBM GB/s vs peak"
HBM_PEAK_GBPS = 8000.0
POLICIES = {"lru": 0, "rotary": 1}  # MOE_POLICY_LRU, MOE_POLICY_ROTARY


def parse():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None,
                    help="timed decode steps (tokens); default 2048 (config 5: 512)")
    ap.add_argument("--warmup", type=int, default=64, help="untimed decode steps before timing")
    ap.add_argument("--config", type=int, default=4, choices=[2, 3, 4, 5],
                    help="4: 40-layer budgeted stack (default); 5: 48-layer int4 prefill + decode; "
                         "2/3: one all-resident layer")
    ap.add_argument("--tokens", type=int, default=1, help="tokens per decode step (config 3)")
    ap.add_argument("--host-alias", action="store_true",
                    help="let every layer read layer 0's host copy (keys stay distinct; same PCIe traffic)")
    ap.add_argument("--cpu-seconds", type=float, default=15.0, help="budget of the oracle CPU baseline")
    ap.add_argument("--prefetch", type=int, default=0,
                    help="speculative prefetch per layer (most often demanded non-resident experts of the next "
                         "layer); 0 = off, the LRU residency the workload specifies")
    ap.add_argument("--policy", choices=["lru", "rotary"], default="lru",
                    help="replacement policy of the expert slots (the workloads specify LRU)")
    ap.add_argument("--charge-max", type=int, default=32, help="rotary policy: most charge a slot holds")
    ap.add_argument("--residency", choices=["host", "device"], default="device",
                    help="where the slot table's decisions are made: lookup kernels (the default: no host round "
                         "trip), or the host after each layer's ids reach it (needed by --prefetch / --recall); "
                         "the decisions are the same")
    ap.add_argument("--attention", action="store_true",
                    help="config 4 shapes with a decoder self-attention block before each MoE block (32 query / 4 "
                         "key-value heads of 128, bf16 KV cache of --context positions; the timed tokens are the "
                         "cache's last positions)")
    ap.add_argument("--context", type=int, default=4096, help="attention: positions of the KV cache")
    ap.add_argument("--graph", action="store_true",
                    help="with device residency, replay each token as one captured HIP graph "
                         "(moe_stack_decode_graph) instead of enqueueing its launches")
    ap.add_argument("--recall", type=int, default=0,
                    help="reverse rotation: remembered tokens whose slot sets a recurring layer-0 routing recalls "
                         "(0 = off)")
    ap.add_argument("--recall-overlap", type=int, default=0,
                    help="layer-0 experts a recalled token must share (0 = all k)")
    ap.add_argument("--routing", choices=["zipf_overlap", "topics"], default="zipf_overlap",
                    help="config 4 routing: the specified Zipf(1.1) 70%% overlap, or recurring contexts "
                         "(--topics contexts, a token keeps its context with --topic-stay)")
    ap.add_argument("--topics", type=int, default=8)
    ap.add_argument("--topic-stay", type=float, default=0.9)
    ap.add_argument("--host-quota", type=int, default=0,
                    help="host tier: per lookup, up to this many non-resident experts computed on host cores from "
                         "the pinned store instead of filled over the link (the layer's previous host share first); "
                         "0 = off")
    ap.add_argument("--host-layers", type=int, default=0,
                    help="host tier: layers below this one computed wholly on host cores (the paper's n-cpu-moe "
                         "recipe); 0 = off")
    ap.add_argument("--host-threads", type=int, default=0, help="host tier threads (0 = every core)")
    ap.add_argument("--replays", type=int, default=5,
                    help="replays of the last step's launches (one per layer) for the per-launch device time")
    return ap.parse_args()


def decoder(torch, stack, xs, bias, graph: bool):
    """One decode token through the stack: the eager step, or (device residency, one token) the step's
    captured graph replayed through fixed buffers -- the token's hidden state and routing mask copied in and
    its output copied back, all inside the timed region."""
    if not graph:
        return lambda tag, t: stack.decode_step(tag, xs[t], None if bias is None else bias[t])
    x_buf = torch.empty_like(xs[0])
    b_buf = None if bias is None else torch.empty_like(bias[0])

    def step(tag, t):
        x_buf.copy_(xs[t])
        if b_buf is not None:
            b_buf.copy_(bias[t])
        stack.decode_graph(tag, x_buf, b_buf)
        xs[t].copy_(x_buf)
    return step


def pcie_ceiling_gbps(torch, moe, chunk: int, total: int) -> float:
    """hipMemcpyAsync of `chunk`-byte pieces from hipHostMalloc memory to the device, back to back
    on one stream (the path the expert cache's fills take)."""
    import ctypes as C
    hip = C.CDLL("libamdhip64.so")
    hip.hipMemcpyAsync.argtypes = [C.c_void_p, C.c_void_p, C.c_size_t, C.c_int, C.c_void_p]
    hip.hipMemcpyAsync.restype = C.c_int
    n = total // chunk
    src = moe.PinnedBuffer(n * chunk)
    src.array[:] = 1
    dst = torch.empty(n * chunk, dtype=torch.uint8, device="cuda")
    st = torch.cuda.Stream()
    best = 0.0
    for _ in range(3):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record(st)
        for i in range(n):
            rc = hip.hipMemcpyAsync(dst.data_ptr() + i * chunk, src.ptr + i * chunk, chunk, 1, st.cuda_stream)
            if rc != 0:
                raise RuntimeError(f"hipMemcpyAsync failed ({rc})")
        b.record(st)
        b.synchronize()
        best = max(best, n * chunk / (a.elapsed_time(b) * 1e-3) / 1e9)
    del dst
    src.close()
    return best


def hbm_ceiling(torch, moe, launch_sizes, n_launch: int = 40, stream_bytes: int = 4 << 30):
    """HBM read rate of the library's streaming probe (the expert kernels' 16-byte nontemporal loads):
    one pass over `stream_bytes`, and `n_launch` groups of back-to-back launches of `launch_sizes` bytes
    (the expert FFN's two launches) over distinct memory (so the 256 MB last-level cache cannot serve
    repeats), replayed from a graph so that host launch cost is out of the picture.  Also runs one 256 MiB
    device copy: the known-size kernels the HBM byte counters are calibrated against."""
    sizes = [int(b) // 16 * 16 for b in launch_sizes]
    launch_bytes = sum(sizes)
    total = max(stream_bytes, launch_bytes * n_launch)
    buf = torch.zeros(total, dtype=torch.uint8, device="cuda")
    sink = torch.zeros(1, dtype=torch.float32, device="cuda")
    cp_src = torch.ones(256 << 20, dtype=torch.uint8, device="cuda")
    cp_dst = torch.empty_like(cp_src)
    cp_dst.copy_(cp_src)
    ev = lambda: torch.cuda.Event(enable_timing=True)
    best_stream = 0.0
    for _ in range(3):
        a, b = ev(), ev()
        a.record()
        moe.moe_hbm_read_probe(buf[:stream_bytes], sink)
        b.record()
        b.synchronize()
        best_stream = max(best_stream, stream_bytes / (a.elapsed_time(b) * 1e-3) / 1e9)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for i in range(n_launch):
            off = i * launch_bytes
            for b in sizes:
                moe.moe_hbm_read_probe(buf[off:off + b], sink)
                off += b
    g.replay()
    torch.cuda.synchronize()
    a, b = ev(), ev()
    reps = 5
    a.record()
    for _ in range(reps):
        g.replay()
    b.record()
    b.synchronize()
    us = a.elapsed_time(b) * 1e3 / (reps * n_launch)
    del g, buf, cp_src, cp_dst
    return {"stream_GBps": best_stream, "stream_bytes": stream_bytes,
            "launch_GBps": launch_bytes / (us * 1e-6) / 1e9, "launch_us": us, "launch_bytes": launch_bytes,
            "method": f"moe_hbm_read_probe: one {stream_bytes >> 30} GiB pass; {n_launch} groups of launches of "
                      f"{'+'.join(str(b) for b in sizes)} B over distinct memory replayed from a graph"}


TRAFFIC_FILES = {4: os.path.join(ROOT, "profiles", "cfg4_expert_ffn_hbm_traffic.txt"),
                 5: os.path.join(ROOT, "profiles", "cfg5_expert_ffn_hbm_traffic.txt")}
CSRC = os.path.join(ROOT, "paper_2605_29135_amd", "csrc")
FFN_KERNELS = ("gateup_kernel", "down_combine_lds_kernel")


def kernel_source(src: str, name: str) -> str:
    """The source text of one kernel template (from its `template` line to its closing brace)."""
    i0 = src.index(f"void {name}(")
    i0 = src.rindex("template", 0, i0)
    return src[i0:src.index("\n}\n", i0) + 3]


def ffn_source_hash() -> str:
    """sha256 of the expert FFN kernels' own source text and of the device helpers they use."""
    import hashlib
    with open(os.path.join(CSRC, "kernels.hip")) as fh:
        src = fh.read()
    h = hashlib.sha256()
    for name in FFN_KERNELS:
        h.update(kernel_source(src, name).encode())
    for helper in ("device_common.h", "residency_dev.h"):
        with open(os.path.join(CSRC, helper), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def measured_traffic(cfg=4):
    """HBM bytes per launch of the gate/up and of the down + combine kernel from the committed counter
    summary (FETCH_SIZE and WRITE_SIZE passes, each calibrated by a known-size kernel): a dict, or None when
    the kernels' source changed since the counters were taken."""
    path = TRAFFIC_FILES[cfg]
    if not os.path.exists(path):
        return None, "no counter summary"
    kv = {}
    with open(path) as fh:
        for line in fh:
            if ":" in line and not line.startswith("#"):
                key, val = line.split(":", 1)
                kv[key.strip()] = val.strip()
    if kv.get("kernel_source_sha256") != ffn_source_hash():
        return None, "kernel source changed since the counters were taken"
    return {"gateup": float(kv["gateup_hbm_bytes_per_launch"]), "down": float(kv["down_hbm_bytes_per_launch"]),
            "gateup_alg": float(kv["gateup_algorithmic_bytes"]), "down_alg": float(kv["down_algorithmic_bytes"])}, \
        path[len(ROOT) + 1:]


def ffn_roofline(gu_bytes, dn_bytes, ktimes, hbm, traffic, traffic_src, replays, n_launch, label):
    """The expert FFN's HBM roofline: algorithmic bytes of its two launches (gate/up + SwiGLU, down +
    combine) over their device time per layer, with each launch's own figure beside it."""
    gu_s, dn_s, ffn_s = ktimes["gateup"] * 1e-3, ktimes["down"] * 1e-3, ktimes["ffn"] * 1e-3
    ffn_bytes = gu_bytes + dn_bytes
    ach = ffn_bytes / ffn_s / 1e9
    if traffic is not None and (abs(traffic["gateup_alg"] - gu_bytes) > 0.01 * gu_bytes or
                                abs(traffic["down_alg"] - dn_bytes) > 0.01 * dn_bytes):
        # the counters were taken on launches of another size (e.g. every rank on the GPU, where a host tier
        # leaves the GPU only its share)
        traffic, traffic_src = None, (f"counters taken on launches of {traffic['gateup_alg']:.0f} + "
                                      f"{traffic['down_alg']:.0f} B; these move {gu_bytes:.0f} + {dn_bytes:.0f} B")
    tr = None if traffic is None else traffic["gateup"] + traffic["down"]
    sub = lambda b, t, tb: {"achieved": b / t / 1e9, "frac": b / t / 1e9 / HBM_PEAK_GBPS, "bytes_per_launch": b,
                            "mean_launch_us": t * 1e6, "traffic": tb,
                            "traffic_over_algorithmic": None if tb is None else tb / b}
    return {"bound": "hbm", "kernel": f"expert FFN ({label}): gate/up + SwiGLU, then down + combine",
            "achieved": ach, "peak": HBM_PEAK_GBPS, "unit": "GB/s", "frac": ach / HBM_PEAK_GBPS,
            "traffic": tr, "traffic_over_algorithmic": None if tr is None else tr / ffn_bytes,
            "traffic_source": traffic_src, "bytes_per_launch": ffn_bytes, "mean_launch_us": ffn_s * 1e6,
            "timing": f"the last step's {n_launch} layers' gate/up and down launches (same arguments, every expert "
                      f"resident: the replays fill nothing, while a budgeted step's own gate/up launch also streams "
                      f"its misses) in one HIP graph, replayed {replays}x between HIP events; per layer"
                      + (f"; the graph repeats the layers' launches {-(-32 // n_launch)}x (at least 32 launches), "
                         f"repeat r reading experts (e + r) mod E of the step's experts e when every expert is "
                         f"resident" if n_launch < 32 else ""),
            "practical_ceiling_GBps": hbm["launch_GBps"], "frac_of_practical": ach / hbm["launch_GBps"],
            "gateup": sub(gu_bytes, gu_s, None if traffic is None else traffic["gateup"]),
            "down": sub(dn_bytes, dn_s, None if traffic is None else traffic["down"])}


def hit_step_ms(torch, dec, xs, t_last, reps=16):
    """Device time of one decode token whose every expert is resident: the last timed token's routing
    replayed (its experts were just used, so every lookup hits), from copies of its input, after the timed
    region.  This is the step's compute with no fill on its path."""
    x_save = xs[t_last].clone()
    dec(t_last + 1, t_last)  # warm, and sets the token's experts most recent
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for i in range(reps):
        xs[t_last].copy_(x_save)
        dec(t_last + 2 + i, t_last)
    torch.cuda.synchronize()
    ms = (time.perf_counter() - t0) * 1e3 / reps
    xs[t_last].copy_(x_save)
    return ms


def link_overlap(d, elapsed, steps, compute_ms, ceil_gbps):
    """Stall and overlap of the demand fills over the timed region, per token: copy = the link's busy time, as
    the filled bytes over the link's measured ceiling; compute = a step whose experts are all resident
    (hit_step_ms); stall = wall - compute (the time the step spent waiting for the link); overlap =
    1 - (wall - max(copy, compute)) / min(copy, compute)."""
    wall = elapsed * 1e3 / steps
    copy = d["h2d_bytes"] / (ceil_gbps * 1e9) * 1e3 / steps
    lo = min(copy, compute_ms)
    return {"stall_ms_per_token": max(0.0, wall - compute_ms), "copy_ms_per_token": copy,
            "compute_ms_per_token": compute_ms, "wall_ms_per_token": wall,
            "overlap": 1.0 - (wall - max(copy, compute_ms)) / lo if lo > 0 else None,
            "method": "copy: filled bytes / the link's measured ceiling; compute: 16 steps repeating the last token's "
                      "routing after the timed region (every expert resident, no fill); stall = wall - compute"}


def clocked_fills(torch, moe, make_stack, dec_factory, n_tokens, first, warmup=64):
    """The demand fills timed on the device (MOE_CACHE_FILL_CLOCK) in a separate run of `n_tokens` decode tokens
    on a fresh cache (after `warmup` untimed ones): the stamps cost each filling launch and lookup a few
    microseconds, so this run is not the timed one."""
    cache, stack = make_stack()
    dec = dec_factory(stack)
    for t in range(first, first + warmup):
        dec(10_000_000 + t, t)
    moe.moe_sync_check()
    s0 = cache.stats()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for t in range(first + warmup, first + warmup + n_tokens):
        dec(10_000_000 + t, t)
    torch.cuda.synchronize()
    el = time.perf_counter() - t0
    moe.moe_sync_check()
    s1 = cache.stats()
    stack.close()
    cache.close()
    fill = (s1["fill_ns"] - s0["fill_ns"]) * 1e-6 / n_tokens
    return {"tokens": n_tokens, "tokens_per_s": n_tokens / el, "wall_ms_per_token": el * 1e3 / n_tokens,
            "fill_ms_per_token": fill, "link_GBps_while_filling":
                (s1["h2d_bytes"] - s0["h2d_bytes"]) / n_tokens / (fill * 1e-3) / 1e9 if fill else None,
            "fill_tail_ms_per_token": (s1["stall_ns"] - s0["stall_ns"]) * 1e-6 / n_tokens,
            "method": "device wall-clock stamps of each filling launch: first to last filling block (fill), and how "
                      "long the fills ran past the launch's computing blocks (fill_tail, the library's stall_ns)"}


def expert_kernel_bytes(wl, n_exp, T):
    """Algorithmic bytes of one gate/up launch and one down + combine launch: the weights of the n_exp
    experts read once (int4: packed nibbles plus bf16 group scales), x read, the activations written and
    read back, the output row read and written."""
    import synth
    H, I, k = wl.H, wl.I, wl.k
    if wl.dtype == synth.INT4G128:
        gu_w, dn_w = 2 * I * H // 2 + 2 * I * (H // 128) * 2, H * I // 2 + H * (I // 128) * 2
    else:
        es = 4 if wl.dtype == synth.F32 else 2
        gu_w, dn_w = 2 * I * H * es, H * I * es
    rows = T * k + (T if wl.shared else 0)
    return n_exp * gu_w + T * H * 4 + rows * I * 4, n_exp * dn_w + rows * I * 4 + T * H * 8


def replay_fills(moe, ev, L, E, capacity, policy, charge_max=0):
    """Fills a host-simulated cache of the library makes when the demand trace `ev` (hit and miss events,
    in order) is looked up again step by step under another replacement policy (placeholder 256-byte blobs:
    the decisions do not depend on the bytes)."""
    eb = 256
    host = np.zeros(L * E * eb, np.uint8)
    c = moe.ExpertCache(L, E, eb, capacity * eb, host.ctypes.data, E * eb, eb, host_sim=True, policy=policy,
                        charge_max=charge_max)
    step_key = ev["t"].astype(np.int64) * 1_000_000 + ev["layer"]
    starts = np.r_[np.flatnonzero(np.r_[True, step_key[1:] != step_key[:-1]]), ev.size]
    for a, b in zip(starts[:-1], starts[1:]):
        c.lookup(int(ev["t"][a]), int(ev["layer"][a]), ev["expert"][a:b])
        c.release()
    fills = c.stats()["misses"]
    c.close()
    return int(fills)


def residency_bound(moe, cache, E, capacity, step_bytes_per_token=None, policy="lru"):
    """The run's fills over its whole demand trace (every lookup from the cold cache on), the same trace
    replayed under each replacement policy of the library (host simulation), and the fewest fills any
    policy could make on it (moe_opt_fills)."""
    ev = cache.trace()
    # prefetched experts that a later demand lookup found resident
    n_pf, used, pending = int((ev["kind"] == moe.EVENT_PREFETCH).sum()), 0, set()
    if n_pf:
        for t_, layer, ex, kind, _, victim in ev.tolist():
            if victim >= 0:
                pending.discard(victim)
            kk = layer * E + ex
            if kind == moe.EVENT_PREFETCH:
                pending.add(kk)
            elif kind == moe.EVENT_HIT and kk in pending:
                used += 1
                pending.discard(kk)
    ev = ev[ev["kind"] != moe.EVENT_PREFETCH]
    if ev.size == 0:
        return None
    keys = (ev["layer"].astype(np.int64) * E + ev["expert"]).astype(np.int32)
    step_key = ev["t"].astype(np.int64) * 1_000_000 + ev["layer"]
    starts = np.flatnonzero(np.r_[True, step_key[1:] != step_key[:-1]])
    offsets = np.r_[starts, ev.size].astype(np.int32)
    n_keys = int(ev["layer"].max() + 1) * E
    L = int(ev["layer"].max() + 1)
    opt = moe.moe_opt_fills_flat(keys, offsets, n_keys, capacity)
    run_fills = int((ev["kind"] == moe.EVENT_MISS).sum())
    # the run's own misses are plain LRU's only when nothing was prefetched; otherwise replay the demand trace
    lru = run_fills if (policy == "lru" and n_pf == 0) else replay_fills(moe, ev, L, E, capacity, moe.MOE_POLICY_LRU)
    rotary = {str(q): replay_fills(moe, ev, L, E, capacity, moe.MOE_POLICY_ROTARY, q) for q in (0, 4, 32)}
    out = {"scope": "every lookup of the run from a cold cache (warm-up included)", "lookups": int(ev.size),
           "run_policy": policy, "run_demand_fills": run_fills,
           "lru_fills": lru, "rotary_fills_by_charge_max": rotary, "opt_fills": int(opt),
           "opt_over_lru": opt / lru if lru else None,
           "rotary32_over_lru": rotary["32"] / lru if lru else None}
    if n_pf:
        out["prefetch_fills"] = n_pf
        out["prefetches_used"] = used  # demanded again before being evicted
    return out


def attention_kernel_line(att, H, ms, n_steps):
    """The attention block's time per layer (its five launches at the last decode position) and the bytes it
    must move: the QKV and output projection weights, and the keys and values of every position it reads."""
    nh, nkv, hd = att["n_heads"], att["n_kv"], att["head_dim"]
    n_pos = att["start_pos"] + n_steps
    w_bytes = 2 * ((nh + 2 * nkv) * hd * H + H * nh * hd)
    kv_bytes = 2 * 2 * n_pos * nkv * hd
    return {"attention_us": ms * 1e3, "attention_bytes_per_layer": w_bytes + kv_bytes,
            "attention_GBps": (w_bytes + kv_bytes) / (ms * 1e-3) / 1e9, "attention_positions": n_pos}


def cpu_baseline(wl, store, steps, bias_np, x_np, budget_s, shared=None, attention=None):
    """The oracle on the host cores: whole tokens through every layer, no budget.  attention(l, t, x) -> x,
    when given, is each layer's attention block before its MoE block."""
    import oracle
    import synth
    routers = [synth.router_weights(wl, l) for l in range(wl.L)]
    t0 = time.perf_counter()
    outs = []
    for i, t in enumerate(steps):
        x = x_np[t].astype(np.float64)
        for l in range(wl.L):
            if attention is not None:
                x = attention(l, t, x)
            h = oracle.rmsnorm(x.astype(np.float32)).astype(np.float32)
            z = oracle.router_logits(h, routers[l], wl.router_dtype) + bias_np[t, l]
            ids, w, _ = oracle.topk_softmax(z.astype(np.float32), wl.k)
            x = x + oracle.moe_ffn(h, ids, w, store(l), wl.H, wl.I, wl.dtype, None if shared is None else shared[l])
        outs.append(x)
        if time.perf_counter() - t0 > budget_s:
            break
    dt = time.perf_counter() - t0
    return len(outs) / dt, outs, dt


def cpu_baseline_line(wl, store, steps, bias_np, x_np, budget_s, bytes_per_token, shared=None, attention=None):
    """The oracle timed on every host core it is given, then on one thread (a third of the budget, at least
    one token); returns the bench line's cpu_baseline object and the all-core run's outputs."""
    import oracle
    cores = oracle.threads_used()
    tps, outs, dt = cpu_baseline(wl, store, steps, bias_np, x_np, budget_s, shared, attention)
    oracle.set_threads(1)
    try:
        tps1, outs1, dt1 = cpu_baseline(wl, store, steps, bias_np, x_np, budget_s / 3, shared, attention)
    finally:
        oracle.set_threads(cores)
    line = {"value": round(tps, 4), "unit": "tokens/s", "cores": cores, "kind": "oracle",
            "cpu_model": oracle.cpu_model(), "GBps": tps * bytes_per_token / 1e9,
            "sample": f"{len(outs)} timed tokens x {wl.L} layers, fp64 C oracle, no budget ({dt:.1f} s)",
            "single_thread": {"value": round(tps1, 4), "unit": "tokens/s", "cores": 1,
                              "GBps": tps1 * bytes_per_token / 1e9,
                              "sample": f"{len(outs1)} timed tokens x {wl.L} layers ({dt1:.1f} s)"}}
    return line, outs


def prefill_ffn_time(torch, moe, synth, wl, layer_blob, shared_blob, router, reps=10):
    """Device time of one layer's expert FFN over the prompt chunk (moe_prefill_grouped: grouping, grouped
    GEMMs, combine) with that layer's experts resident, routed by its router; events around `reps` calls."""
    x = torch.from_numpy(synth.prefill_states(wl)).cuda()
    h = torch.empty_like(x)
    _, ids, w = moe.moe_route_topk(x, router, wl.router_dtype, wl.k, rmsnorm=True, x_norm=h)
    ws = torch.empty(moe.moe_prefill_workspace_bytes(wl.prefill, wl.k, wl.E, wl.H, wl.I), dtype=torch.uint8,
                     device="cuda")
    y = torch.empty_like(x)
    call = lambda: moe.moe_prefill_grouped(h, ids, w, layer_blob, wl.expert_bytes, wl.dtype, wl.I, wl.E,
                                           shared_w=shared_blob, y_out=y, workspace=ws)
    call()
    torch.cuda.synchronize()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record()
    for _ in range(reps):
        call()
    b.record()
    b.synchronize()
    moe.moe_sync_check()
    return a.elapsed_time(b) / reps


def run_prefill_decode(args, torch, moe, oracle, synth):
    """Config 5: a prompt chunk, then batch-1 decode, through 48 int4 layers under the 6 GiB budget."""
    wl = synth.workload(5)
    L, E, k, H, I, eb, Tp = wl.L, wl.E, wl.k, wl.H, wl.I, wl.expert_bytes, wl.prefill
    steps = wl.steps if args.steps is None else args.steps
    n_steps = args.warmup + steps
    dev = torch.device("cuda:0")
    t_setup = time.perf_counter()
    buf = moe.PinnedBuffer(L * E * eb)
    store = buf.array.reshape(L, E, eb)
    synth.fill_host_store(wl, buf.array)
    routers = [torch.from_numpy(synth.router_weights(wl, l)).to(dev) for l in range(L)]
    shared_np = [synth.expert_blob(wl, l, None) for l in range(L)]
    shared = [torch.from_numpy(b).to(dev) for b in shared_np]
    sets = synth.routing_sets(wl, steps=n_steps)
    bias_np = np.zeros((n_steps, L, 1, E), np.float32)
    for t in range(n_steps):
        for l in range(L):
            bias_np[t, l] = synth.mask_logits(wl, sets[t, l])
    x_np = np.stack([synth.hidden_states(wl, t) for t in range(n_steps)])
    xs = torch.from_numpy(x_np).to(dev)
    bias = torch.from_numpy(bias_np).to(dev)
    xp_np = synth.prefill_states(wl)
    t_setup = time.perf_counter() - t_setup

    def make(fill_clock=False):
        cache = moe.ExpertCache(L, E, eb, wl.budget_bytes, buf.ptr, E * eb, eb, reserved_bytes=L * eb,
                                policy=POLICIES[args.policy], charge_max=args.charge_max,
                                device=args.residency == "device", fill_clock=fill_clock)
        stack = moe.MoeStack(cache, H, I, E, k, wl.dtype, wl.router_dtype, routers, shared, max_tokens=1,
                             max_prefill_tokens=Tp, prefetch=args.prefetch)
        return cache, stack

    # warm-up on a throw-away cache (kernels loaded, allocator warm), so the timed run starts cold
    use_graph = args.residency == "device" and args.graph
    cache, stack = make()
    stack.prefill(0, torch.from_numpy(xp_np[:64]).to(dev))
    dec = decoder(torch, stack, xs, bias, use_graph)
    for t in range(min(args.warmup, 8)):
        dec(1 + t, t)
    moe.moe_sync_check()
    stack.close()
    cache.close()
    torch.cuda.synchronize()

    cache, stack = make()
    xp = torch.from_numpy(xp_np).to(dev)
    st0 = cache.stats()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    stack.prefill(0, xp)
    torch.cuda.synchronize()
    t_prefill = time.perf_counter() - t0
    moe.moe_sync_check()
    st1 = cache.stats()
    dec = decoder(torch, stack, xs, bias, use_graph)
    run = lambda a, b: [dec(1 + t, t) for t in range(a, b)]
    run(0, args.warmup)
    moe.moe_sync_check()
    st2 = cache.stats()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    run(args.warmup, n_steps)
    torch.cuda.synchronize()
    t_decode = time.perf_counter() - t0
    moe.moe_sync_check()
    st3 = cache.stats()
    compute_ms = hit_step_ms(torch, dec, xs, n_steps - 1)
    clocked = None
    if args.residency == "device" and n_steps >= 96:
        xs_c = xs.clone()  # the clocked run works on its own copy of the inputs
        clocked = clocked_fills(torch, moe, lambda: make(fill_clock=True),
                                lambda st: decoder(torch, st, xs_c, bias, use_graph), min(256, n_steps - 64), 0)
        del xs_c
    ktimes = {name: stack.kernel_time(w, args.replays) for w, name in enumerate(["route", "gateup", "down", "ffn"])}
    moe.moe_sync_check()
    bound = residency_bound(moe, cache, E, st3["capacity"], policy=args.policy)
    stack.close()
    cache.close()

    tok_s = steps / t_decode
    gu_bytes, dn_bytes = expert_kernel_bytes(wl, k + 1, 1)
    hbm = hbm_ceiling(torch, moe, [gu_bytes, dn_bytes])
    traffic, traffic_src = measured_traffic(5)
    roof = ffn_roofline(gu_bytes, dn_bytes, ktimes, hbm, traffic, traffic_src, args.replays, L, "int4 decode")

    # the prompt chunk's expert FFN on the matrix cores, one layer with its experts resident
    layer_blob = torch.from_numpy(np.ascontiguousarray(store[L - 1]).reshape(-1)).to(dev)
    pf_ms = prefill_ffn_time(torch, moe, synth, wl, layer_blob, shared[L - 1], routers[L - 1])
    del layer_blob
    rows = Tp * k + Tp
    pf_flop = 2.0 * rows * (2 * I) * H + 2.0 * rows * H * I

    d_pf = {f: st1[f] - st0[f] for f in ("lookups", "hits", "misses", "evictions", "prefetches", "h2d_bytes")}
    d_dec = {f: st3[f] - st2[f] for f in ("lookups", "hits", "misses", "evictions", "h2d_bytes", "stall_ns",
                                          "fill_ns")}
    ceil = max(pcie_ceiling_gbps(torch, moe, eb, 256 * eb), pcie_ceiling_gbps(torch, moe, 64 << 20, 1 << 30))
    h2d_tok = d_dec["h2d_bytes"] / steps

    sample = list(range(args.warmup, n_steps))
    cpu_line, outs = cpu_baseline_line(wl, lambda l: store[l], sample, bias_np, x_np, args.cpu_seconds,
                                       L * (k + 1) * eb + L * wl.router_bytes, shared=shared_np)
    gpu_x = xs[sample[0]:sample[0] + len(outs)].cpu().numpy().astype(np.float64)
    err = 0.0
    for i, o in enumerate(outs):
        delta_ref = o - x_np[sample[i]]
        delta = gpu_x[i] - x_np[sample[i]]
        err = max(err, float(np.abs(delta - delta_ref).max() / np.abs(delta_ref).max()))
    out = {
        "metric": METRIC,
        "value": round(tok_s, 3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": steps,
        "warmup": args.warmup,
        "ms_per_step": round(t_decode * 1e3 / steps, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": synth.DTYPE_NAMES[wl.dtype],
        "data": "synthetic (seeded N(0,0.02) weights quantised to int4 g128, N(0,1) hidden states, "
                "router-chosen prefill routing, Zipf-overlap decode routing masks)",
        "config": {"workload": wl.name, "layers": L, "experts": E, "top_k": k, "shared_expert": True,
                   "hidden": H, "intermediate": I, "prefill_tokens": Tp, "decode_tokens_per_step": 1,
                   "budget_bytes": wl.budget_bytes, "slots": st3["capacity"], "host_store_bytes": L * E * eb,
                   "prefetch_per_layer": args.prefetch, "policy": args.policy, "residency": args.residency,
                   "decode_graph": use_graph,
                   **({"charge_max": args.charge_max} if args.policy == "rotary" else {})},
        "roofline": roof,
        "hbm_ceiling": hbm,
        "kernels": {"route_us": ktimes["route"] * 1e3, "gateup_us": ktimes["gateup"] * 1e3,
                    "down_us": ktimes["down"] * 1e3, "ffn_us": ktimes["ffn"] * 1e3},
        "prefill": {"tokens": Tp, "tokens_per_s": Tp / t_prefill, "ms": t_prefill * 1e3,
                    "h2d_bytes": d_pf["h2d_bytes"], "misses": d_pf["misses"],
                    "prefetches": d_pf["prefetches"],
                    "h2d_GBps": d_pf["h2d_bytes"] / t_prefill / 1e9,
                    "layer_ffn_ms": pf_ms, "layer_ffn_flop": pf_flop,
                    "roofline": {"bound": "mfma", "kernel": "one layer's prompt-chunk expert FFN (grouping, "
                                 "grouped bf16 MFMA GEMMs, combine)", "achieved": pf_flop / (pf_ms * 1e-3) / 1e12,
                                 "peak": 2500.0, "unit": "TFLOP/s",
                                 "frac": pf_flop / (pf_ms * 1e-3) / 1e12 / 2500.0}},
        "residency": {**d_dec, "miss_rate": d_dec["misses"] / d_dec["lookups"] if d_dec["lookups"] else 0.0,
                      "misses_per_token": d_dec["misses"] / steps, "bound": bound},
        "pcie": {"h2d_bytes_per_token": h2d_tok, "achieved_GBps": d_dec["h2d_bytes"] / t_decode / 1e9,
                 "ceiling_GBps": ceil, "frac": d_dec["h2d_bytes"] / t_decode / 1e9 / ceil,
                 "tokens_per_s_bound": ceil * 1e9 / h2d_tok if h2d_tok else None,
                 **(link_overlap(d_dec, t_decode, steps, compute_ms, ceil) if args.residency == "device" else {}),
                 "clocked_fills": clocked},
        "cpu_baseline": cpu_line,
        "parity": {"sampled_tokens": len(outs), "max_normwise_err": err},
        "setup_s": round(t_setup, 1),
        "paper_context": "21.06 decode tokens/s and 74.2 prompt tokens/s at ~6.3 GB VRAM, RTX 4060 Laptop 8 GB, "
                         "Qwen3.6-35B-A3B Q4_K_M",
    }
    print(json.dumps(out))


def main():
    args = parse()
    if (args.prefetch or args.recall or args.host_quota or args.host_layers) and args.residency == "device":
        args.residency = "host"  # prefetch, recall and the host tier decide on the host
    if args.gpus != 1:
        print(f"bench.py measures one GPU: the library has no multi-GPU path (asked for --gpus {args.gpus})",
              file=sys.stderr)
        sys.exit(2)
    import torch

    import oracle
    import paper_2605_29135_amd as moe
    import synth

    torch.cuda.set_device(0)
    moe.moe_init(0)
    if args.config == 5:
        return run_prefill_decode(args, torch, moe, oracle, synth)
    if args.steps is None:
        args.steps = 2048
    dev = torch.device("cuda:0")
    T = args.tokens
    if args.config == 4 and args.routing == "topics":
        wl = synth.workload(4, routing="topics", topics=args.topics, topic_stay=args.topic_stay,
                            name=f"cfg4 shapes with recurring contexts: 40-layer bf16 H2048 E128 k8 I768, 6 GiB, "
                                 f"{args.topics} contexts, stay {args.topic_stay}, keep 0.85")
    elif args.config == 4:
        wl = synth.workload(4)
    else:
        wl = synth.workload(args.config, T=T)
    L, E, k, H, I, eb = wl.L, wl.E, wl.k, wl.H, wl.I, wl.expert_bytes
    budgeted = wl.budget_bytes is not None
    n_steps = args.warmup + args.steps

    # ---- inputs: host expert store, routers, routing masks, hidden states
    t_setup = time.perf_counter()
    alias = args.host_alias and L > 1
    L_store = 1 if alias else L
    buf = moe.PinnedBuffer(L_store * E * eb)
    store = buf.array.reshape(L_store, E, eb)
    if alias:
        synth.layer_experts(wl, 0, store[0])
    else:
        synth.fill_host_store(wl, buf.array)
    routers = [torch.from_numpy(synth.router_weights(wl, l)).to(dev) for l in range(L)]
    shared = [torch.from_numpy(synth.expert_blob(wl, l, None)).to(dev) for l in range(L)] if wl.shared else None
    if wl.routing == "router":
        bias_np = None
    else:
        sets = synth.routing_sets(wl, steps=n_steps, T=T)
        bias_np = np.zeros((n_steps, L, T, E), np.float32)
        for t in range(n_steps):
            for l in range(L):
                bias_np[t, l] = synth.mask_logits(wl, sets[t, l])
    x_np = np.stack([synth.hidden_states(wl, t, T=T) for t in range(n_steps)])
    xs = torch.from_numpy(x_np).to(dev)
    bias = None if bias_np is None else torch.from_numpy(bias_np).to(dev)
    reserved = L * eb if wl.shared else 0
    budget = wl.budget_bytes if budgeted else L * E * eb + reserved
    def make_cache(fill_clock=False):
        return moe.ExpertCache(L, E, eb, budget, buf.ptr, 0 if alias else E * eb, eb, reserved_bytes=reserved,
                               preload=not budgeted, policy=POLICIES[args.policy], charge_max=args.charge_max,
                               device=budgeted and args.residency == "device",
                               host_layers=args.host_layers if budgeted else 0,
                               host_quota=args.host_quota if budgeted else 0, fill_clock=fill_clock)
    cache = make_cache()
    hybrid = budgeted and (args.host_layers > 0 or args.host_quota > 0)
    att = None
    if args.attention:
        # synthetic, seeded: N(0, 0.02) projection weights, an N(0, 1) cache prefix; the timed tokens take the
        # cache's last positions
        nh, nkv, hd, max_pos = 32, 4, 128, args.context
        start = max_pos - n_steps
        if start < 0:
            raise SystemExit(f"--context {max_pos} is shorter than the {n_steps} decode steps")
        gen = torch.Generator(device=dev)
        att = dict(n_heads=nh, n_kv=nkv, head_dim=hd, max_pos=max_pos, theta=1.0e6, start_pos=start,
                   w_qkv=[], w_o=[], k_cache=[], v_cache=[])
        for l in range(L):
            gen.manual_seed(7000 + l)
            rnd = lambda *shape, sd=1.0: (torch.randn(*shape, generator=gen, device=dev) * sd).to(torch.bfloat16)
            att["w_qkv"].append(rnd((nh + 2 * nkv) * hd, H, sd=0.02).view(torch.int16))
            att["w_o"].append(rnd(H, nh * hd, sd=0.02).view(torch.int16))
            att["k_cache"].append(rnd(nkv, hd // 8, max_pos, 8).view(torch.int16))
            att["v_cache"].append(rnd(nkv, max_pos, hd).view(torch.int16))
        torch.cuda.synchronize()
    stack = moe.MoeStack(cache, H, I, E, k, wl.dtype, wl.router_dtype, routers, shared, max_tokens=T,
                         prefetch=args.prefetch if budgeted else 0, recall=args.recall if budgeted else 0,
                         recall_overlap=args.recall_overlap, attention=att, host_threads=args.host_threads)
    t_setup = time.perf_counter() - t_setup

    stream = torch.cuda.current_stream()

    use_graph = budgeted and args.residency == "device" and T == 1 and args.graph
    dec = decoder(torch, stack, xs, bias, use_graph)

    def run(t0, t1):
        for t in range(t0, t1):
            dec(t, t)

    # ---- warm-up, then the timed region
    run(0, args.warmup)
    moe.moe_sync_check(stream)
    st0 = cache.stats()
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    run(args.warmup, n_steps)
    torch.cuda.synchronize()
    elapsed = time.perf_counter() - t0
    moe.moe_sync_check(stream)
    st1 = cache.stats()
    compute_ms = hit_step_ms(torch, dec, xs, n_steps - 1) if budgeted and att is None else None
    clocked = None
    if budgeted and args.residency == "device" and att is None and not hybrid and T == 1 and n_steps >= 96:
        def make_clocked():
            c = make_cache(fill_clock=True)
            return c, moe.MoeStack(c, H, I, E, k, wl.dtype, wl.router_dtype, routers, shared, max_tokens=T)
        xs_c = xs.clone()  # the clocked run works on its own copy of the inputs
        clocked = clocked_fills(torch, moe, make_clocked, lambda st: decoder(torch, st, xs_c, bias, use_graph),
                                min(256, n_steps - 64), 0)
        del xs_c
    # the oracle leg's copy of the attention state, taken before the attention timing rewrites the last position
    att_host = None
    if att is not None:
        att_host = dict(wq=[t.cpu().numpy().view(np.uint16) for t in att["w_qkv"]],
                        wo=[t.cpu().numpy().view(np.uint16) for t in att["w_o"]],
                        kc=[moe.key_cache_plain(t.cpu().numpy().view(np.uint16)) for t in att["k_cache"]],
                        vc=[t.cpu().numpy().view(np.uint16) for t in att["v_cache"]])
    # per-launch device time: each kernel of the last layer re-launched back to back between two events
    ktimes = {name: stack.kernel_time(w, args.replays) for w, name in enumerate(["route", "gateup", "down", "ffn"])}
    if att is not None:
        ktimes["attention"] = stack.kernel_time(4, args.replays)
    if not budgeted and L < 32:  # the same expert FFN re-reading the step's own experts in every repeat
        ktimes["ffn_same_experts"] = stack.kernel_time(8 + 3, args.replays)
    moe.moe_sync_check(stream)

    tok_s = args.steps * T / elapsed
    ms_step = elapsed * 1e3 / args.steps

    # ---- roofline of the dominant kernel (expert gate/up + SwiGLU)
    unique = k if T == 1 else None
    if unique is None:
        unique = float(np.mean([len(np.unique(sets[t, 0])) for t in range(args.warmup, n_steps)]))
    if hybrid:  # the timing re-launches skip the ranks the host tier computed in the last step
        ev_all = cache.trace()
        last = ev_all[ev_all["t"] == ev_all["t"].max()]
        unique = k - float((last["kind"] == moe.EVENT_HOST).sum()) / L
    n_exp = unique + (1 if wl.shared else 0)
    gu_bytes, dn_bytes = expert_kernel_bytes(wl, n_exp, T)

    # ---- residency and PCIe
    d = {f: st1[f] - st0[f] for f in ("lookups", "hits", "misses", "evictions", "h2d_bytes", "stall_ns", "fill_ns",
                                      "host_computed")}
    h2d_per_tok = d["h2d_bytes"] / (args.steps * T)
    pcie = None
    if budgeted:
        ceil_expert = pcie_ceiling_gbps(torch, moe, eb, 128 * eb)
        ceil_large = pcie_ceiling_gbps(torch, moe, 64 << 20, 1 << 30)
        ceil = max(ceil_expert, ceil_large)
        pcie = {"h2d_bytes_per_token": h2d_per_tok, "achieved_GBps": d["h2d_bytes"] / elapsed / 1e9,
                "ceiling_GBps": ceil, "ceiling_expert_chunks_GBps": ceil_expert,
                "frac": d["h2d_bytes"] / elapsed / 1e9 / ceil,
                "tokens_per_s_bound": ceil * 1e9 / h2d_per_tok if h2d_per_tok else None,
                "ceiling_method": "hipMemcpyAsync from hipHostMalloc memory, 64 MiB and expert-size chunks",
                **(link_overlap(d, elapsed, args.steps, compute_ms, ceil) if compute_ms and args.residency == "device"
                   else {}), "clocked_fills": clocked}

    hbm = hbm_ceiling(torch, moe, [gu_bytes, dn_bytes])
    traffic, traffic_src = measured_traffic(4) if args.config == 4 else (None, "no counter summary")
    roof = ffn_roofline(gu_bytes, dn_bytes, ktimes, hbm, traffic, traffic_src, args.replays, L,
                        f"{synth.DTYPE_NAMES[wl.dtype]} decode, T={T}")
    if "ffn_same_experts" in ktimes:
        ach_same = (gu_bytes + dn_bytes) / (ktimes["ffn_same_experts"] * 1e-3) / 1e9
        roof["same_experts_every_launch"] = {
            "achieved": ach_same, "frac": ach_same / HBM_PEAK_GBPS, "mean_launch_us": ktimes["ffn_same_experts"] * 1e3,
            "note": "every repeat re-reads the step's own experts, which the last-level cache may then hold"}

    bound = residency_bound(moe, cache, E, st1["capacity"], policy=args.policy) if budgeted and not hybrid else None
    host_tier = None
    if hybrid:
        hb = d["host_computed"] * eb
        host_tier = {"host_layers": args.host_layers, "host_quota": args.host_quota,
                     "threads": args.host_threads or len(os.sched_getaffinity(0)),
                     "experts_per_token": d["host_computed"] / (args.steps * T),
                     "bytes_per_token": hb / (args.steps * T), "achieved_GBps": hb / elapsed / 1e9,
                     "note": "experts computed on host cores from the pinned store (not filled); achieved_GBps is "
                             "their weight bytes over the timed wall time"}

    # ---- oracle on the host cores (bounded sample of the timed tokens), with a parity check
    sample = list(range(args.warmup, n_steps))
    att_hook = None
    if att_host is not None:
        att_hook = lambda l, t, x: oracle.attention_decode(x.astype(np.float32), att_host["wq"][l], att_host["wo"][l],
                                                           att_host["kc"][l], att_host["vc"][l], att["start_pos"] + t,
                                                           att["n_heads"], att["n_kv"], theta=att["theta"])
    cpu_bytes = L * T * (n_exp * eb + wl.router_bytes)
    cpu_line, outs = cpu_baseline_line(wl, lambda l: store[0 if alias else l], sample, bias_np
                                       if bias_np is not None else np.zeros((n_steps, L, T, E), np.float32),
                                       x_np, args.cpu_seconds, cpu_bytes,
                                       shared=[synth.expert_blob(wl, l, None) for l in range(L)] if wl.shared
                                       else None, attention=att_hook)
    gpu_x = xs[sample[0]:sample[0] + len(outs)].cpu().numpy().astype(np.float64)
    err = 0.0
    for i, o in enumerate(outs):
        delta_ref = o - x_np[sample[i]]
        delta = gpu_x[i] - x_np[sample[i]]
        err = max(err, float(np.abs(delta - delta_ref).max() / np.abs(delta_ref).max()))

    wl_name = wl.name if T == 1 else f"{wl.name} (T={T})"
    if hybrid:
        wl_name = (f"{wl_name}; with a host tier (host_layers {args.host_layers}, host_quota {args.host_quota}: those "
                   f"experts computed on host cores from the pinned store)")
    if att is not None:
        wl_name = (f"{wl_name}; with a decoder self-attention block per layer ({att['n_heads']}/{att['n_kv']} heads "
                   f"of {att['head_dim']}, positions {att['start_pos']}..{att['start_pos'] + n_steps - 1} of a "
                   f"{att['max_pos']}-position bf16 KV cache)")
    out = {
        "metric": METRIC,
        "value": round(tok_s, 3),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": synth.DTYPE_NAMES[wl.dtype],
        "data": "synthetic (seeded N(0,0.02) weights, N(0,1) hidden states, Zipf-overlap routing masks)",
        "config": {"workload": wl_name, "layers": L, "experts": E, "top_k": k, "hidden": H, "intermediate": I,
                   "tokens_per_step": T, "budget_bytes": budget, "slots": st1["capacity"],
                   "host_store_bytes": L_store * E * eb, "host_layers_aliased": bool(alias),
                   "prefetch_per_layer": args.prefetch if budgeted else 0, "policy": args.policy,
                   "residency": args.residency if budgeted else "preloaded", "decode_graph": use_graph,
                   **({"charge_max": args.charge_max} if args.policy == "rotary" else {}),
                   **({"recall": args.recall, "recall_overlap": args.recall_overlap or k} if args.recall else {}),
                   **({"attention": {"n_heads": att["n_heads"], "n_kv": att["n_kv"], "head_dim": att["head_dim"],
                                     "kv_positions": att["max_pos"], "first_position": att["start_pos"]}}
                      if att is not None else {})},
        "roofline": roof,
        "hbm_ceiling": hbm,
        "kernels": {"route_us": ktimes["route"] * 1e3, "gateup_us": ktimes["gateup"] * 1e3,
                    "down_us": ktimes["down"] * 1e3, "ffn_us": ktimes["ffn"] * 1e3,
                    **(attention_kernel_line(att, H, ktimes["attention"], n_steps) if att is not None else {})},
        "residency": {**d, "miss_rate": d["misses"] / d["lookups"] if d["lookups"] else 0.0,
                      "misses_per_token": d["misses"] / (args.steps * T), "bound": bound},
        "pcie": pcie,
        **({"host_tier": host_tier} if host_tier else {}),
        "cpu_baseline": cpu_line,
        "parity": {"sampled_tokens": len(outs), "max_normwise_err": err},
        "setup_s": round(t_setup, 1),
        "paper_context": "21.06 decode tokens/s at ~6.3 GB VRAM, RTX 4060 Laptop 8 GB, Qwen3.6-35B-A3B Q4_K_M",
    }
    print(json.dumps(out))


if __name__ == "__main__":
    main()
