"""Benchmark of the fused RoPE + causal attention hot path on one MI355X.

Default workload: the Llama-3-8B attention layer (B=1, H=32, H_kv=8, S=8192,
D=128, bf16, NeoX RoPE theta=500000, causal).  One step = the fused forward
plus the three-kernel backward on one batch of synthetic N(0,1) inputs that
are already resident in HBM.  `value` is the algorithmic (causal-effective)
TFLOP/s of that step: 4*D flops per visible (query, key) pair forward and
10*D backward.

Alongside, on the same inputs and outside the timed steps:
* per-call durations from HIP events (fused forward, backward, rotation,
  separate forward) and the roofline of the fused forward kernel;
* the separate-RoPE path (rotation kernel, then the forward without RoPE) and
  the rotation kernel's HBM bandwidth, measured over a buffer pool larger than
  twice the 256 MB Infinity Cache;
* the fuse-vs-separate crossover over S = 1024..16384 (skip with --no-sweep),
  each figure the GPU time per call from HIP-graph replays (median of 20
  replays of 10 captured calls; the rotation over its whole pool), and the rotation
  calculus model fitted to it (crossover_model: fused extra time a*S^2,
  separate rotation b*S, model crossover b/a next to the measured one);
* decode over a KV cache at the paper's three decode geometries (skip with
  --no-decode): GPU time per call from HIP-graph replays (and the eager
  per-call median beside it) and cache bandwidth against the HBM peak, the
  caches rotated through a pool larger than twice the Infinity Cache;
* block-sparse attention with a BigBird-style mask at N = 4096 (skip with
  --no-sparse): forward and backward medians, TFLOP/s over the visible pairs,
  and the dense forward of the same shape for the speedup;
* the other attention workloads at full size (skip with --no-workloads): the
  sliding-window (W = 1024, GQA) and ALiBi + causal shapes and the D = 64
  RoPE + causal shape, each forward and backward (median of 50 and 20 calls
  after 10 and 3 warm-ups) against the MFMA peak, and, with RoPE, the
  separate path (rotation + no-RoPE forward) next to the fused forward;
* the paper's RoPE comparison rows (skip with --no-variants): fused vs
  separate RoPE for no mask, causal and a 256-key sliding window at B=4,
  H=12, D=64, S = 512..4096, timed like the sweep; and the dense-bias and
  relu extensions' forward and backward at B=4, H=16, S=4096, D=128;
* a plain device-to-device copy of 512 MiB: the achievable HBM bandwidth next
  to the rotation kernel's, and the calibration kernel for the HBM-traffic
  counters;
* the fp64 CPU oracle timed on a bounded sample (cpu_baseline).

roofline.traffic is the forward kernel's measured HBM bytes per launch,
taken from profiles/fwd_llama3_8b_hbm_traffic.json, which records the hash of
the kernel sources it was measured on; if the sources differ, it is null.

Prints ONE JSON line.  Only --gpus 1 is supported.
"""
import argparse
import functools
import json
import math
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2516.6     # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0         # MI355X HBM3E
# The paper's decode latencies on H100 (Table tab:decode), other hardware: context only.
PAPER_DECODE_MS = {"decode_llama3_8b_h32kv8_cache4096": 0.034, "decode_llama3_70b_h64kv8_cache32768": 0.184,
                   "decode_mistral_7b_h32kv8_cache16384": 0.072}
# The paper's block-sparse forward latency (BigBird mask, N = 4096), other hardware: context only.
PAPER_SPARSE_MS = {"bigbird_b4h12s4096d64": 0.084}
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "fwd_llama3_8b_hbm_traffic.json")
FWD_SOURCES = ("fwd_bf16.hip", "attn_tiles.hpp", "common.hpp")


def fwd_source_hash():
    import hashlib
    h = hashlib.sha256()
    for name in FWD_SOURCES:
        with open(os.path.join(ROOT, "paper_2609_13612_amd", "csrc", name), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def measured_traffic(workload):
    """HBM bytes per fused-forward launch from the committed counter summary, if current."""
    try:
        with open(TRAFFIC_FILE) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None
    if rec.get("workload") != workload or rec.get("source_sha256") != fwd_source_hash():
        return None
    return rec.get("traffic_bytes_per_launch")


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def crossover_fit(sweep, w, s_min=4096, rows_per_rotation=256):
    """Fit the rotation-calculus model to the sweep (Section 5.3, Eq. 1 restated
    with consistent units): the fused kernel's extra time over the no-RoPE
    kernel grows as a * S^2 (every workgroup of `rows_per_rotation` query rows
    rotates each K tile it visits once), the separate rotation as b * S (one HBM
    round trip of Q and K).  Fitted by least squares through the origin on the
    points with S >= s_min, where both kernels fill the GPU; the model's
    crossover is S* = b / a.  Also reported: the measured crossover (where the
    fused speedup crosses 1, interpolated in log S), the fused kernel's
    effective cost per rotated K element, the VALU operations per element that
    cost stands for at the chip's fp32 lane rate (e_rot * (1 - phi)), and the
    rotation's achieved bandwidth."""
    pts = [r for r in sweep if r["S"] >= s_min]
    if len(pts) < 2:
        return None
    a = sum((r["fused_ms"] - r["norope_ms"]) * r["S"] ** 2 for r in pts) / sum(r["S"] ** 4 for r in pts)
    b = sum(r["rope_ms"] * r["S"] for r in pts) / sum(r["S"] ** 2 for r in pts)
    measured = None
    for lo, hi in zip(sweep, sweep[1:]):
        if (lo["fused_speedup"] - 1.0) * (hi["fused_speedup"] - 1.0) <= 0 and lo["fused_speedup"] != hi["fused_speedup"]:
            f = (lo["fused_speedup"] - 1.0) / (lo["fused_speedup"] - hi["fused_speedup"])
            measured = round(math.exp(math.log(lo["S"]) + f * (math.log(hi["S"]) - math.log(lo["S"]))))
            break
    # rotated K elements per fused launch at S: B*H*S^2*D / (2 * rows_per_rotation) (causal)
    rot_elems_per_s2 = w.B * w.H * w.D / (2.0 * rows_per_rotation)
    c_rot_s = a * 1e-3 / rot_elems_per_s2            # seconds per rotated element
    lane_rate = 256 * 4 * 16 * 2.4e9                  # fp32 VALU lane operations per second
    bytes_per_s = 4.0 * w.B * (w.H + w.Hkv) * w.D     # separate rotation bytes per unit S
    return {"fit_points_S": [r["S"] for r in pts],
            "a_ms_per_S2": a, "b_ms_per_S": b,
            "S_star_model": round(b / a) if a > 0 else None,
            "S_star_measured": measured,
            "fused_rot_ps_per_element": round(c_rot_s * 1e12, 3),
            "e_rot_times_1_minus_phi": round(c_rot_s * lane_rate, 2),
            "rotation_gbs_fit": round(bytes_per_s / (b * 1e-3) / 1e9, 1),
            "rows_per_rotation": rows_per_rotation}


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="llama3_8b_b1h32kv8s8192d128")
    ap.add_argument("--no-sweep", action="store_true", help="skip the fuse-vs-separate sweep over S")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-decode", action="store_true", help="skip the decode (KV-cache) measurements")
    ap.add_argument("--no-sparse", action="store_true", help="skip the block-sparse (BigBird mask) measurements")
    ap.add_argument("--no-workloads", action="store_true", help="skip the other attention workloads")
    ap.add_argument("--no-variants", action="store_true",
                    help="skip the RoPE mask variants (paper geometry) and the bias / relu extensions")
    ap.add_argument("--seed", type=int, default=0)
    return ap.parse_args()


def main():
    args = parse()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU path (--gpus must be 1)", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2609_13612_amd import api, blockmask, inputs
    from paper_2609_13612_amd.workloads import DECODE_WORKLOADS, LLAMA_SWEEP_S, SPARSE_WORKLOADS, WORKLOADS

    w = WORKLOADS[args.workload]
    torch.cuda.set_device(0)
    dev = torch.device("cuda:0")
    log(f"workload {w.name}: B={w.B} H={w.H} Hkv={w.Hkv} S={w.S} D={w.D} rope={w.rope} mask={w.mask}")
    cpu = inputs.make_qkv(w.B, w.H, w.Hkv, w.S, w.D, seed=args.seed, with_do=True)
    q, k, v, do = (cpu[n].to(dev) for n in ("q", "k", "v", "do"))
    slopes = inputs.alibi_slopes(w.H).to(dev) if w.alibi else None
    kw = dict(rope=w.rope, theta=w.theta, mask=w.mask, window=w.window or None, alibi_slopes=slopes)
    o = torch.empty_like(q)
    lse = torch.empty(w.B, w.H, w.S, device=dev, dtype=torch.float32)
    dq, dk, dv = torch.empty_like(q), torch.empty_like(k), torch.empty_like(v)
    ws = torch.empty(api.attnfuse_bwd_workspace_bytes(w.B, w.H, w.Hkv, w.S, w.D, w.rope), device=dev, dtype=torch.uint8)
    do_bwd = w.backward

    def step(ev=None):
        if ev is not None:
            ev[0].record()
        api.attnfuse_fwd(q, k, v, out=o, lse=lse, **kw)
        if ev is not None:
            ev[1].record()
        if do_bwd:
            api.attnfuse_bwd(q, k, v, o, do, lse, dq=dq, dk=dk, dv=dv, workspace=ws, **kw)
            if ev is not None:
                ev[2].record()

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    log(f"warmup done ({args.warmup} steps)")

    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(args.steps)]
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0.record()
    for i in range(args.steps):
        step(evs[i])
    t1.record()
    torch.cuda.synchronize()
    total_ms = t0.elapsed_time(t1)
    ms_step = total_ms / args.steps
    fwd_ms = [e[0].elapsed_time(e[1]) for e in evs]
    bwd_ms = [e[1].elapsed_time(e[2]) for e in evs] if do_bwd else []
    log(f"timed {args.steps} steps: {ms_step:.3f} ms/step")

    fwd_flops = w.fwd_flops()
    bwd_flops = w.bwd_flops() if do_bwd else 0
    step_flops = fwd_flops + bwd_flops
    value = step_flops / (ms_step * 1e-3) / 1e12
    fwd_avg = statistics.mean(fwd_ms)
    fwd_tf = fwd_flops / (fwd_avg * 1e-3) / 1e12
    result_extra = {
        "fwd": {"ms_avg": round(fwd_avg, 4), "ms_median": round(statistics.median(fwd_ms), 4),
                "tflops": round(fwd_tf, 1), "frac_peak": round(fwd_tf / PEAK_BF16_TFLOPS, 4),
                "flops": fwd_flops},
    }
    if do_bwd:
        bwd_avg = statistics.mean(bwd_ms)
        bwd_tf = bwd_flops / (bwd_avg * 1e-3) / 1e12
        result_extra["bwd"] = {"ms_avg": round(bwd_avg, 4), "ms_median": round(statistics.median(bwd_ms), 4),
                               "tflops": round(bwd_tf, 1), "frac_peak": round(bwd_tf / PEAK_BF16_TFLOPS, 4),
                               "flops": bwd_flops, "kernels": 3}

    # ---------------------------------------------------------------- separate-RoPE path
    def time_calls(fn, reps):
        es = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(reps)]
        for a, b in es:
            a.record()
            fn()
            b.record()
        torch.cuda.synchronize()
        return [a.elapsed_time(b) for a, b in es]

    graph_failures = []

    def graph_call_ms(fns, reps=20):
        """GPU time per call of a sequence of calls with no host work between them: the calls are
        captured once into a HIP graph and the graph is replayed; median replay time / len(fns).
        Below about 20 us per call the eager figures measure the binding's host overhead instead.
        If the capture fails, the eager per-call median is returned and the failure is reported
        in the JSON line (graph_timing_failures)."""
        g = torch.cuda.CUDAGraph()
        torch.cuda.synchronize()
        try:
            with torch.cuda.graph(g):
                for fn in fns:
                    fn()
        except RuntimeError as e:
            torch.cuda.synchronize()
            graph_failures.append(str(e).splitlines()[0][:200])
            log(f"graph capture failed ({graph_failures[-1]}); eager timing instead")
            return statistics.median(time_calls(lambda: [fn() for fn in fns], reps)) / len(fns)
        torch.cuda.synchronize()
        for _ in range(3):
            g.replay()
        es = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(reps)]
        for a, b in es:
            a.record()
            g.replay()
            b.record()
        torch.cuda.synchronize()
        ms = statistics.median(a.elapsed_time(b) for a, b in es) / len(fns)
        del g
        return ms

    separate = None
    rope_bw = None
    if w.rope != "none":
        nbytes = w.rope_bytes()
        npool = max(2, math.ceil(600e6 / nbytes))
        pool = [(q.clone(), k.clone()) for _ in range(npool)]
        outs = [(torch.empty_like(q), torch.empty_like(k)) for _ in range(npool)]
        it = [0]

        def rot():
            i = it[0] % npool
            it[0] += 1
            api.attnfuse_rope(pool[i][0], pool[i][1], rope=w.rope, theta=w.theta, out_q=outs[i][0], out_k=outs[i][1])

        for _ in range(3):
            rot()
        rot_ms = time_calls(rot, 4 * npool)
        rot_avg = statistics.mean(rot_ms)
        rope_bw = nbytes / (rot_avg * 1e-3) / 1e9
        qr, kr = outs[0]
        kw_none = dict(kw, rope="none")

        def sep_fwd():
            api.attnfuse_fwd(qr, kr, v, out=o, lse=lse, **kw_none)

        sep_ms = time_calls(sep_fwd, max(10, args.steps))
        sep_avg = statistics.mean(sep_ms)
        separate = {"rope_ms_avg": round(rot_avg, 4), "fwd_norope_ms_avg": round(sep_avg, 4),
                    "total_ms": round(rot_avg + sep_avg, 4),
                    "fused_speedup": round((rot_avg + sep_avg) / fwd_avg, 4),
                    "rope_bytes": nbytes, "rope_gbs": round(rope_bw, 1),
                    "rope_frac_hbm_peak": round(rope_bw / PEAK_HBM_GBS, 4), "rope_buffer_pool": npool}
        del pool, outs
        log(f"separate path: rope {rot_avg:.4f} ms ({rope_bw:.0f} GB/s) + fwd {sep_avg:.4f} ms")

    sweep = None
    crossover = None
    if not args.no_sweep and w.rope != "none":
        sweep = []
        for S in LLAMA_SWEEP_S:
            c = inputs.make_qkv(w.B, w.H, w.Hkv, S, w.D, seed=args.seed)
            qs, ks, vs = (c[n].to(dev) for n in ("q", "k", "v"))
            os_ = torch.empty_like(qs)
            ls = torch.empty(w.B, w.H, S, device=dev, dtype=torch.float32)
            nb = w.rope_bytes(S)
            npool = max(2, math.ceil(600e6 / nb))
            pq = [(qs.clone(), ks.clone()) for _ in range(npool)]
            po = [(torch.empty_like(qs), torch.empty_like(ks)) for _ in range(npool)]
            rots = [functools.partial(api.attnfuse_rope, pq[i][0], pq[i][1], rope=w.rope, theta=w.theta,
                                      out_q=po[i][0], out_k=po[i][1]) for i in range(npool)]

            def fused_s():
                api.attnfuse_fwd(qs, ks, vs, out=os_, lse=ls, **kw)

            def none_s():
                api.attnfuse_fwd(po[0][0], po[0][1], vs, out=os_, lse=ls, **dict(kw, rope="none"))

            for fn in rots + [fused_s] * 10 + [none_s] * 10:
                fn()
            r_ms = graph_call_ms(rots)
            f_ms = graph_call_ms([fused_s] * 10)
            n_ms = graph_call_ms([none_s] * 10)
            sweep.append({"S": S, "fused_ms": round(f_ms, 4), "rope_ms": round(r_ms, 4), "norope_ms": round(n_ms, 4),
                          "fused_speedup": round((r_ms + n_ms) / f_ms, 4),
                          "fused_tflops": round(w.fwd_flops(S) / (f_ms * 1e-3) / 1e12, 1)})
            log(f"sweep S={S}: fused {f_ms:.4f} ms, rope {r_ms:.4f} + norope {n_ms:.4f} ms")
            del pq, po, qs, ks, vs, os_, ls
        torch.cuda.empty_cache()
        crossover = crossover_fit(sweep, w)

    # ---------------------------------------------------------------- plain copy reference
    copy_bytes = 512 << 20
    src = torch.empty(copy_bytes, device=dev, dtype=torch.uint8)
    dst = torch.empty_like(src)
    dst.copy_(src)
    cp_ms = statistics.median(time_calls(lambda: dst.copy_(src), 10))
    copy_gbs = 2 * copy_bytes / (cp_ms * 1e-3) / 1e9
    del src, dst
    log(f"plain copy of 512 MiB: {cp_ms:.4f} ms, {copy_gbs:.0f} GB/s moved")

    # ---------------------------------------------------------------- decode over a KV cache
    decode = None
    if not args.no_decode:
        decode = {}
        for name, dw in DECODE_WORKLOADS.items():
            c = inputs.make_decode(dw.B, dw.H, dw.Hkv, dw.S_kv, dw.D, seed=args.seed)
            qd = c["q"].to(dev)
            nb = dw.cache_bytes()
            npool = max(2, math.ceil(600e6 / nb))   # more than twice the Infinity Cache: HBM, not MALL
            kv_pool = [(c["k"].to(dev), c["v"].to(dev)) for _ in range(npool)]
            del c
            od = torch.empty_like(qd)
            ld = torch.empty(dw.B, dw.H, device=dev, dtype=torch.float32)
            wsd = torch.empty(api.attnfuse_decode_workspace_bytes(dw.B, dw.H, dw.Hkv, dw.S_kv, dw.D),
                              device=dev, dtype=torch.uint8)
            cnt = [0]

            def dec():
                i = cnt[0] % npool
                cnt[0] += 1
                api.attnfuse_decode(qd, kv_pool[i][0], kv_pool[i][1], rope=dw.rope, theta=dw.theta, out=od,
                                    lse=ld, workspace=wsd)

            for _ in range(10):
                dec()
            # GPU time per call (graph replays over the cache pool); the eager figure adds the
            # binding's host overhead, which is comparable to a call's ~10-30 us of GPU work
            d_eager = statistics.median(time_calls(dec, max(50, 2 * npool)))
            d_ms = graph_call_ms([functools.partial(api.attnfuse_decode, qd, kv_pool[i][0], kv_pool[i][1], rope=dw.rope,
                                                    theta=dw.theta, out=od, lse=ld, workspace=wsd)
                                  for i in range(npool)])
            gbs = nb / (d_ms * 1e-3) / 1e9
            decode[name] = {"B": dw.B, "H": dw.H, "H_kv": dw.Hkv, "S_kv": dw.S_kv, "D": dw.D, "rope": dw.rope,
                            "ms": round(d_ms, 4), "ms_eager": round(d_eager, 4), "cache_bytes": nb,
                            "roofline": {"bound": "hbm", "achieved": round(gbs, 1), "peak": PEAK_HBM_GBS,
                                         "unit": "GB/s", "frac": round(gbs / PEAK_HBM_GBS, 4)},
                            "frac_of_copy": round(gbs / copy_gbs, 4), "cache_pool": npool,
                            "paper_h100_ms": PAPER_DECODE_MS.get(name)}
            log(f"decode {name}: {d_ms:.4f} ms, {gbs:.0f} GB/s of cache (eager calls {d_eager:.4f} ms)")
            del kv_pool, qd, od, ld, wsd
        torch.cuda.empty_cache()

    # ---------------------------------------------------------------- block-sparse attention
    sparse = None
    if not args.no_sparse:
        sparse = {}
        for name, sw in SPARSE_WORKLOADS.items():
            c = inputs.make_qkv(sw.B, sw.H, sw.Hkv, sw.S, sw.D, seed=args.seed, with_do=True)
            qb, kb, vb, dob = (c[n].to(dev) for n in ("q", "k", "v", "do"))
            del c
            active = sw.active()
            bm = blockmask.block_mask_from_dense(torch.from_numpy(active), sw.S, device=dev)
            ob, lb = torch.empty_like(qb), torch.empty(sw.B, sw.H, sw.S, device=dev, dtype=torch.float32)
            grads = (torch.empty_like(qb), torch.empty_like(kb), torch.empty_like(vb))
            wsb = torch.empty(api.attnfuse_bwd_workspace_bytes(sw.B, sw.H, sw.Hkv, sw.S, sw.D), device=dev,
                              dtype=torch.uint8)
            skw = dict(rope="none", mask="none")

            def sp_fwd():
                api.attnfuse_fwd_blocksparse(qb, kb, vb, bm, out=ob, lse=lb, **skw)

            def sp_bwd():
                api.attnfuse_bwd_blocksparse(qb, kb, vb, ob, dob, lb, bm, dq=grads[0], dk=grads[1], dv=grads[2],
                                             workspace=wsb, **skw)

            def dense_fwd():
                api.attnfuse_fwd(qb, kb, vb, out=ob, lse=lb, **skw)

            res = {}
            # in this order the backward reads the block-sparse forward's O and LSE
            for label, fn in (("dense_fwd", dense_fwd), ("fwd", sp_fwd), ("bwd", sp_bwd)):
                for _ in range(10):
                    fn()
                res[label] = statistics.median(time_calls(fn, 50))
            f_tf = sw.fwd_flops(active) / (res["fwd"] * 1e-3) / 1e12
            b_tf = sw.bwd_flops(active) / (res["bwd"] * 1e-3) / 1e12
            sparse[name] = {"B": sw.B, "H": sw.H, "H_kv": sw.Hkv, "S": sw.S, "D": sw.D, "block": 64,
                            "active_blocks": int(active.sum()), "density": round(float(active.mean()), 4),
                            "fwd_ms": round(res["fwd"], 4), "fwd_tflops": round(f_tf, 1),
                            "bwd_ms": round(res["bwd"], 4), "bwd_tflops": round(b_tf, 1),
                            "dense_fwd_ms": round(res["dense_fwd"], 4),
                            "fwd_speedup_vs_dense": round(res["dense_fwd"] / res["fwd"], 3),
                            "paper_fwd_ms": PAPER_SPARSE_MS.get(name)}
            log(f"block-sparse {name}: density {active.mean():.4f}, fwd {res['fwd']:.4f} ms ({f_tf:.0f} TF/s), "
                f"bwd {res['bwd']:.4f} ms, dense fwd {res['dense_fwd']:.4f} ms")
            del qb, kb, vb, dob, ob, lb, grads, wsb, bm
        torch.cuda.empty_cache()

    # ---------------------------------------------------------------- the other attention workloads
    others = None
    if not args.no_workloads:
        others = {}
        for name, ow in WORKLOADS.items():
            if name == w.name or ow.S < 1024:   # the headline, and the tiny parity case
                continue
            c = inputs.make_qkv(ow.B, ow.H, ow.Hkv, ow.S, ow.D, seed=args.seed, with_do=True)
            qw, kw_, vw, dow = (c[n].to(dev) for n in ("q", "k", "v", "do"))
            del c
            sl = inputs.alibi_slopes(ow.H).to(dev) if ow.alibi else None
            okw = dict(rope=ow.rope, theta=ow.theta, mask=ow.mask, window=ow.window or None, alibi_slopes=sl)
            ow_o = torch.empty_like(qw)
            ow_l = torch.empty(ow.B, ow.H, ow.S, device=dev, dtype=torch.float32)
            ow_g = (torch.empty_like(qw), torch.empty_like(kw_), torch.empty_like(vw))
            ow_ws = torch.empty(api.attnfuse_bwd_workspace_bytes(ow.B, ow.H, ow.Hkv, ow.S, ow.D, ow.rope),
                                device=dev, dtype=torch.uint8)

            def ofwd():
                api.attnfuse_fwd(qw, kw_, vw, out=ow_o, lse=ow_l, **okw)

            def obwd():
                api.attnfuse_bwd(qw, kw_, vw, ow_o, dow, ow_l, dq=ow_g[0], dk=ow_g[1], dv=ow_g[2], workspace=ow_ws,
                                 **okw)

            for _ in range(10):
                ofwd()
            f_ms = statistics.median(time_calls(ofwd, 50))
            for _ in range(3):
                obwd()
            b_ms = statistics.median(time_calls(obwd, 20))
            f_tf = ow.fwd_flops() / (f_ms * 1e-3) / 1e12
            b_tf = ow.bwd_flops() / (b_ms * 1e-3) / 1e12
            rec = {"B": ow.B, "H": ow.H, "H_kv": ow.Hkv, "S": ow.S, "D": ow.D, "rope": ow.rope, "mask": ow.mask,
                   "window": ow.window, "alibi": ow.alibi,
                   "fwd_ms": round(f_ms, 4), "fwd_tflops": round(f_tf, 1), "fwd_frac_peak": round(f_tf / PEAK_BF16_TFLOPS, 4),
                   "bwd_ms": round(b_ms, 4), "bwd_tflops": round(b_tf, 1), "bwd_frac_peak": round(b_tf / PEAK_BF16_TFLOPS, 4)}
            msg = f"{name}: fwd {f_ms:.4f} ms ({f_tf:.0f} TF/s), bwd {b_ms:.4f} ms ({b_tf:.0f} TF/s)"
            if ow.rope != "none":
                nbytes = ow.rope_bytes()
                npool = max(2, math.ceil(600e6 / nbytes))
                pool = [(qw.clone(), kw_.clone()) for _ in range(npool)]
                outs = [(torch.empty_like(qw), torch.empty_like(kw_)) for _ in range(npool)]
                it2 = [0]

                def orot():
                    i = it2[0] % npool
                    it2[0] += 1
                    api.attnfuse_rope(pool[i][0], pool[i][1], rope=ow.rope, theta=ow.theta, out_q=outs[i][0],
                                      out_k=outs[i][1])

                for _ in range(3):
                    orot()
                r_ms = statistics.median(time_calls(orot, max(20, 2 * npool)))
                qr_, kr_ = outs[0]

                def osep():
                    api.attnfuse_fwd(qr_, kr_, vw, out=ow_o, lse=ow_l, **dict(okw, rope="none"))

                for _ in range(3):
                    osep()
                n_ms = statistics.median(time_calls(osep, 50))
                rec["separate"] = {"rope_ms": round(r_ms, 4), "fwd_norope_ms": round(n_ms, 4),
                                   "total_ms": round(r_ms + n_ms, 4), "fused_speedup": round((r_ms + n_ms) / f_ms, 4),
                                   "rope_gbs": round(nbytes / (r_ms * 1e-3) / 1e9, 1)}
                msg += f"; separate {r_ms + n_ms:.4f} ms (fused speedup {(r_ms + n_ms) / f_ms:.3f})"
                del pool, outs
            others[name] = rec
            log(msg)
            del qw, kw_, vw, dow, ow_o, ow_l, ow_g, ow_ws
        torch.cuda.empty_cache()

    # ---------------------------------------------------------------- RoPE mask variants and extensions
    variants = None
    if not args.no_variants:
        from paper_2609_13612_amd.workloads import Workload
        variants = {"rope_masks": {}, "extensions": {}}
        # Fused vs rotate-then-attend for RoPE + Dense / Causal / SW (W = 256) on the GPT-2-small heads
        # of the paper's variant comparison (B = 4, H = 12, D = 64), N = 512 .. 4096.
        for mask, window in (("none", 0), ("causal", 0), ("sliding_window", 256)):
            for S in (512, 1024, 2048, 4096):
                vw = Workload(f"v_{mask}_{S}", 4, 12, 12, S, 64, rope="neox", theta=10000.0, mask=mask, window=window)
                c = inputs.make_qkv(vw.B, vw.H, vw.Hkv, S, vw.D, seed=args.seed)
                qv, kv_, vv = (c[n].to(dev) for n in ("q", "k", "v"))
                del c
                vkw = dict(theta=vw.theta, mask=mask, window=window or None)
                vo = torch.empty_like(qv)
                vl = torch.empty(vw.B, vw.H, S, device=dev, dtype=torch.float32)

                def vfused():
                    api.attnfuse_fwd(qv, kv_, vv, out=vo, lse=vl, rope="neox", **vkw)

                nb = vw.rope_bytes()
                npool = max(2, math.ceil(600e6 / nb))
                vpool = [(qv.clone(), kv_.clone()) for _ in range(npool)]
                vouts = [(torch.empty_like(qv), torch.empty_like(kv_)) for _ in range(npool)]
                vrots = [functools.partial(api.attnfuse_rope, vpool[i][0], vpool[i][1], rope="neox", theta=vw.theta,
                                           out_q=vouts[i][0], out_k=vouts[i][1]) for i in range(npool)]
                qr_, kr_ = vouts[0]

                def vplain():
                    api.attnfuse_fwd(qr_, kr_, vv, out=vo, lse=vl, rope="none", **vkw)

                res = {}
                for label, fns in (("fused", [vfused] * 20), ("rope", vrots), ("plain", [vplain] * 20)):
                    for fn in fns[:10]:
                        fn()
                    res[label] = graph_call_ms(fns)
                sep = res["rope"] + res["plain"]
                f_tf = vw.fwd_flops() / (res["fused"] * 1e-3) / 1e12
                variants["rope_masks"][f"{mask}_n{S}"] = {
                    "B": vw.B, "H": vw.H, "S": S, "D": vw.D, "mask": mask, "window": window,
                    "fused_ms": round(res["fused"], 4), "fused_tflops": round(f_tf, 1),
                    "rope_ms": round(res["rope"], 4), "fwd_norope_ms": round(res["plain"], 4),
                    "fused_speedup": round(sep / res["fused"], 4)}
                log(f"RoPE + {mask} N={S}: fused {res['fused']:.4f} ms, separate {sep:.4f} ms "
                    f"(fused speedup {sep / res['fused']:.3f})")
                del qv, kv_, vv, vo, vl, vpool, vouts
        # Dense additive bias (a key-padding bias [B, 1, 1, S], broadcast over heads and queries) and relu
        # attention, forward and backward, with RoPE and the causal mask at B = 4, H = 16, S = 4096, D = 128.
        ew = Workload("ext_b4h16s4096d128", 4, 16, 16, 4096, 128, rope="neox", theta=10000.0, mask="causal")
        c = inputs.make_qkv(ew.B, ew.H, ew.Hkv, ew.S, ew.D, seed=args.seed, with_do=True)
        qe, ke, ve, doe = (c[n].to(dev) for n in ("q", "k", "v", "do"))
        del c
        gen = torch.Generator("cpu").manual_seed(args.seed + 7)
        pad = (torch.rand(ew.B, 1, 1, ew.S, generator=gen) < 0.1).float() * -1e4   # about 10 % of keys padded
        bias = pad.to(dev)
        ekw = dict(rope="neox", theta=ew.theta, mask="causal")
        eg = (torch.empty_like(qe), torch.empty_like(ke), torch.empty_like(ve))
        ews = torch.empty(api.attnfuse_bwd_workspace_bytes(ew.B, ew.H, ew.Hkv, ew.S, ew.D, "neox"), device=dev,
                          dtype=torch.uint8)
        for label, norm, b_ in (("softmax_bias", "softmax", bias), ("relu", "relu", None)):
            eo, el = api.attnfuse_fwd_bias_norm(qe, ke, ve, bias=b_, norm=norm, **ekw)

            def efwd():
                api.attnfuse_fwd_bias_norm(qe, ke, ve, bias=b_, norm=norm, out=eo, lse=el, **ekw)

            def ebwd():
                api.attnfuse_bwd_bias_norm(qe, ke, ve, eo, doe, el, bias=b_, norm=norm, dq=eg[0], dk=eg[1],
                                           dv=eg[2], workspace=ews, **ekw)

            for _ in range(5):
                efwd()
            f_ms = statistics.median(time_calls(efwd, 30))
            for _ in range(3):
                ebwd()
            b_ms = statistics.median(time_calls(ebwd, 10))
            f_tf = ew.fwd_flops() / (f_ms * 1e-3) / 1e12
            b_tf = ew.bwd_flops() / (b_ms * 1e-3) / 1e12
            variants["extensions"][label] = {
                "B": ew.B, "H": ew.H, "S": ew.S, "D": ew.D, "rope": "neox", "mask": "causal",
                "bias": "key padding [B,1,1,S]" if b_ is not None else None, "norm": norm,
                "fwd_ms": round(f_ms, 4), "fwd_tflops": round(f_tf, 1), "fwd_frac_peak": round(f_tf / PEAK_BF16_TFLOPS, 4),
                "bwd_ms": round(b_ms, 4), "bwd_tflops": round(b_tf, 1), "bwd_frac_peak": round(b_tf / PEAK_BF16_TFLOPS, 4)}
            log(f"{label}: fwd {f_ms:.4f} ms ({f_tf:.0f} TF/s), bwd {b_ms:.4f} ms ({b_tf:.0f} TF/s)")
            del eo, el
        # the plain fused forward of the same shape, for reference
        for _ in range(5):
            api.attnfuse_fwd(qe, ke, ve, **ekw)
        p_ms = statistics.median(time_calls(lambda: api.attnfuse_fwd(qe, ke, ve, **ekw), 30))
        variants["extensions"]["plain_fwd_ms"] = round(p_ms, 4)
        del qe, ke, ve, doe, eg, ews, bias, pad
        torch.cuda.empty_cache()

    # ---------------------------------------------------------------- CPU oracle baseline
    cpu_baseline = None
    if not args.no_cpu_baseline:
        import numpy as np
        import threadpoolctl
        import oracle
        # the thread count is set explicitly for the BLAS numpy uses (the host's
        # share of cores: OMP_NUM_THREADS where the machine sets it, else the
        # cores this process may run on), and the count in force is reported
        want = int(os.environ.get("OMP_NUM_THREADS") or len(os.sched_getaffinity(0)))
        limiter = threadpoolctl.threadpool_limits(limits=want, user_api="blas")
        blas = [p for p in threadpoolctl.threadpool_info() if p.get("user_api") == "blas"]
        cores = max((p["num_threads"] for p in blas), default=1)
        G = w.H // w.Hkv
        NG = min(3, w.Hkv)        # K/V groups in the sample: about 10-15 s of CPU work at the Llama shape
        f = inputs.to_f64
        sl = slice(0, NG * G)
        okw = dict(rope=w.rope, theta=w.theta, mask=w.mask, window=w.window or None,
                   alibi_slopes=None if slopes is None else f(slopes.cpu())[sl])
        qs, ks, vs, dos = (f(cpu["q"][:1, sl]), f(cpu["k"][:1, :NG]), f(cpu["v"][:1, :NG]), f(cpu["do"][:1, sl]))
        ta = time.perf_counter()
        oracle.attention_forward(qs, ks, vs, **okw)
        if do_bwd:
            oracle.attention_backward(qs, ks, vs, dos, **okw)
        tb = time.perf_counter()
        frac = NG * G / (w.B * w.H)
        sample_flops = (fwd_flops + bwd_flops) * frac
        limiter.restore_original_limits()
        cpu_baseline = {"value": round(sample_flops / (tb - ta) / 1e12, 6), "unit": "TFLOP/s", "cores": cores,
                        "kind": "oracle", "seconds": round(tb - ta, 2),
                        "sample": f"batch 0, query heads 0..{NG * G - 1} with K/V heads 0..{NG - 1} "
                                  f"({NG * G} of {w.B * w.H} heads), "
                                  f"{'forward + backward' if do_bwd else 'forward'}, fp64 numpy, full S={w.S}"}
        log(f"cpu oracle sample: {tb - ta:.1f} s")

    roofline = {"bound": "mfma", "kernel": "fwd_bf16_kernel (fused RoPE + mask, one launch per forward)",
                "achieved": round(fwd_tf, 1), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                "frac": round(fwd_tf / PEAK_BF16_TFLOPS, 4), "traffic": measured_traffic(w.name)}

    line = {
        "metric": "fused RoPE+causal attention TFLOP/s (fwd, bwd) and % of bf16 MFMA peak",
        "value": round(value, 1),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": w.name, "B": w.B, "H": w.H, "H_kv": w.Hkv, "S": w.S, "D": w.D, "rope": w.rope,
                   "rope_theta": w.theta, "mask": w.mask, "window": w.window, "alibi": w.alibi,
                   "step": "fused fwd + bwd" if do_bwd else "fused fwd", "seed": args.seed},
        "frac_peak": round(value / PEAK_BF16_TFLOPS, 4),
        "roofline": roofline,
        "cpu_baseline": cpu_baseline,
        **result_extra,
        "separate_rope": separate,
        "hbm_copy_reference": {"bytes_moved": 2 * copy_bytes, "ms": round(cp_ms, 4), "gbs": round(copy_gbs, 1),
                               "frac_hbm_peak": round(copy_gbs / PEAK_HBM_GBS, 4)},
    }
    if sweep is not None:
        line["crossover_sweep"] = sweep
        line["crossover_model"] = crossover
    if decode is not None:
        line["decode"] = decode
    if sparse is not None:
        line["block_sparse"] = sparse
    if others is not None:
        line["workloads"] = others
    if variants is not None:
        line["variants"] = variants
    if graph_failures:
        line["graph_timing_failures"] = graph_failures
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
