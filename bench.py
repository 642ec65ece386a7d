"""Benchmark of the packed low-bit KV-cache decode path on one MI355X.

One step = one decode token per sequence through the whole hot path:
  1. adapted Q/K/V projection of the B new hidden states (Eq. (1)-(2)),
  2. quantize-and-pack append of the new K/V into the packed cache (for
     window formats such as KIVI the projection call does it:
     kvq_project_append writes the new rows straight into the fp16 window),
  3. decode attention over the in-kernel reconstruction of all cached tokens
     (Hadamard rotation of q and the output where the format rotates).
The cache is first filled to the workload's context with the same kernels
(prefill projection in chunks, then append).  Inputs are synthetic, seeded
and resident in HBM before the timed region.

Timing (HIP events on the launch stream, created without the system-scope
fence that torch's events carry):
  cold   the K timed steps run one after another, each preceded -- outside
         its own events -- by a 1 GiB write that evicts the 256 MB
         Infinity Cache (MALL) and the L2s, so every step streams its
         weights and cache from HBM.  ``value`` is B K / (sum of the K step
         durations), with events only at the step boundaries; a second cold
         pass with events between the calls gives the per-call breakdown
         (``*_marker_events``: each recorded event is a packet of its own,
         about 4 µs on this GPU), and a third times the projection and the
         attention calls with events recorded by their kernels' own
         dispatches (kvq_time_launches: first kernel's start to last
         kernel's end, as a profiler's kernel trace measures them);
         ``roofline`` and the per-call times use the third;
  warm   the same K steps back to back from the same starting cache, with
         nothing in between (the serving loop as it runs): ``warm``.
The K steps are bracketed by a device synchronize on both sides.

Output: one JSON line.  ``value`` is decoded tokens per second (B tokens per
step).  ``roofline`` reports the decode-attention launch (split + merge
kernels): algorithmic bytes per launch (packed codes + fp32 metadata + fp16
window + bf16 q + fp32 o) over its mean cold duration, against MI355X's
8 TB/s HBM peak, with the measured device-to-device copy bandwidth beside
it.  ``per_config`` repeats the measurement (fewer steps) on the other
workloads.  ``cpu_baseline`` times the CPU oracle on a bounded sample of
decode steps, on all host cores and on one.

  python bench.py [--steps K] [--warmup W] [--workload NAME] [--no-cpu-baseline] [--no-per-config]
  python bench.py --phase prefill [--workload gqa12b_b8]   (projection GEMM, MFMA roofline)
  python bench.py --phase merge [--workload llama8b_had]    (dense adapter merge, HBM roofline)
  python bench.py --phase prefill_attn [--workload gqa12b_b8] (chunked prefill attention, MFMA roofline)
  python bench.py --phase append [--workload gqa12b_b8]     (one prefill chunk appended, HBM roofline)
  python bench.py --phase project_append [--workload gqa12b_b8] (projection fused with the append, MFMA roofline)
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import re
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "packed-cache decode attn tokens/s + achieved HBM GB/s (% peak) per config"
HBM_PEAK_GBS = 8000.0
BF16_PEAK_TFLOPS = 2500.0
DEFAULT_WORKLOAD = "llama8b_kivi"
FLUSH_BYTES = 1 << 30       # > 4x the 256 MB MALL
PER_CONFIG_STEPS = 24


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None, help="timed steps (default: the workload's decode steps)")
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default=DEFAULT_WORKLOAD)
    ap.add_argument("--phase", choices=["decode", "prefill", "merge", "prefill_attn", "append", "project_append"],
                    default="decode")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-per-config", action="store_true",
                    help="skip the shorter cold/warm measurement of the other workloads")
    ap.add_argument("--no-warm", action="store_true", help="skip the back-to-back (warm) loop")
    ap.add_argument("--meta-fp16", action="store_true",
                    help="store scales and offsets as fp16 (the paper's storage) instead of the workload's fp32")
    ap.add_argument("--bits8", action="store_true",
                    help="8-bit key and value codes (the 8-bit ablation) in the workload's groups and modes")
    ap.add_argument("--sink", type=int, default=0,
                    help="keep the first SINK tokens as fp16 rows (KVarN's sink tokens; a multiple of 32)")
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="target CPU time of the all-core oracle sample (the one-thread sample is one step)")
    ap.add_argument("--copy-probe-mb", type=int, default=0,
                    help="before the timed region, copy a buffer of this many MiB once (a kernel of known "
                         "bytes for calibrating rocprofv3 FETCH_SIZE/WRITE_SIZE counters)")
    return ap.parse_args()


class FenceFreeEvent:
    """A HIP timing event created with hipEventDisableSystemFence and recorded
    on the current stream.  torch's events carry a system-scope fence (a
    cache writeback and invalidate) at every record, which costs several
    microseconds on this GPU and disturbs the caches of the work that
    follows; the timings of the decode steps use these instead."""
    _lib = None

    def __init__(self, torch):
        import ctypes
        if FenceFreeEvent._lib is None:
            lib = ctypes.CDLL("libamdhip64.so")
            lib.hipEventCreateWithFlags.argtypes = [ctypes.POINTER(ctypes.c_void_p), ctypes.c_uint]
            lib.hipEventRecord.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
            lib.hipEventSynchronize.argtypes = [ctypes.c_void_p]
            lib.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p, ctypes.c_void_p]
            lib.hipEventDestroy.argtypes = [ctypes.c_void_p]
            FenceFreeEvent._lib = lib
        self._torch = torch
        self._ev = ctypes.c_void_p()
        if FenceFreeEvent._lib.hipEventCreateWithFlags(ctypes.byref(self._ev), 0x20000000) != 0:
            raise RuntimeError("hipEventCreateWithFlags failed")

    def record(self):
        if FenceFreeEvent._lib.hipEventRecord(self._ev, self._torch.cuda.current_stream().cuda_stream) != 0:
            raise RuntimeError("hipEventRecord failed")

    @property
    def handle(self) -> int:
        """The hipEvent_t, for kvq_time_launches (recorded by the kernels' own dispatches)."""
        return self._ev.value

    def elapsed_time(self, end) -> float:
        """Milliseconds from this event to `end` (both recorded and complete)."""
        import ctypes
        FenceFreeEvent._lib.hipEventSynchronize(end._ev)
        ms = ctypes.c_float()
        if FenceFreeEvent._lib.hipEventElapsedTime(ctypes.byref(ms), self._ev, end._ev) != 0:
            raise RuntimeError("hipEventElapsedTime failed")
        return ms.value

    def __del__(self):
        if FenceFreeEvent._lib is not None and self._ev:
            FenceFreeEvent._lib.hipEventDestroy(self._ev)


def kernel_source_hash() -> str:
    """Hash of the decode-attention sources (the kernel the traffic counters describe)."""
    import glob
    csrc = os.path.join(ROOT, "paper_2609_04263_amd", "csrc")
    files = sorted(glob.glob(os.path.join(csrc, "attn*.hip")) + glob.glob(os.path.join(csrc, "attn*.h")))
    files += [os.path.join(csrc, f) for f in ("kvq_device.h", "kvq_internal.h")]
    h = hashlib.sha256()
    for f in files:
        with open(f, "rb") as fh:
            h.update(os.path.basename(f).encode())
            h.update(fh.read())
    return h.hexdigest()[:16]


def measured_traffic(workload: str):
    """HBM bytes per launch of the decode-attention kernel from the committed
    rocprofv3 counter summary, or None when it is missing or was taken on a
    different version of the kernel source."""
    path = os.path.join(ROOT, "profiles", f"decode_attn_{workload}_traffic.md")
    if not os.path.exists(path):
        return None
    text = open(path).read()
    src = re.search(r"kernel_source_sha256_16:\s*([0-9a-f]+)", text)
    val = re.search(r"traffic_bytes_per_launch:\s*([0-9.eE+]+)", text)
    if not src or not val or src.group(1) != kernel_source_hash():
        return None
    return float(val.group(1))


def with_variants(wl, args):
    import dataclasses
    if args.meta_fp16:
        wl = dataclasses.replace(wl, name=wl.name + "+meta16", fmt=dict(wl.fmt, meta_fp16=1))
    if args.bits8:
        wl = dataclasses.replace(wl, name=wl.name + "+k8v8", fmt=dict(wl.fmt, k_bits=8, v_bits=8))
    if args.sink:
        wl = dataclasses.replace(wl, name=wl.name + "+sink%d" % args.sink, fmt=dict(wl.fmt, sink=args.sink))
    return wl


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py measures one GPU only (asked for --gpus {args.gpus}, WORLD_SIZE {world}): "
              "the decode path shards over (sequence, KV head) units with no exchange; "
              "multi-GPU runs are not implemented.", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    import __graft_entry__
    __graft_entry__._ensure_built()
    from paper_2609_04263_amd import configs, kvq, synth

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = torch.device("cuda:0")
    wl = with_variants(configs.WORKLOADS[args.workload], args)

    def bf16(bits):
        return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).to(dev).view(torch.bfloat16)

    def alloc_proj(wl, M):
        return (torch.empty((M, wl.d_q), dtype=torch.bfloat16, device=dev),
                torch.empty((M, wl.d_kv), dtype=torch.bfloat16, device=dev),
                torch.empty((M, wl.d_kv), dtype=torch.bfloat16, device=dev),
                torch.empty(max(16, kvq.project_workspace_bytes(M, wl.rank)), dtype=torch.uint8, device=dev))

    if args.phase != "decode":
        W, A, Bm = (bf16(x) for x in synth.layer_weights(wl))
        ap = lambda M: alloc_proj(wl, M)
        if args.phase == "prefill":
            return bench_prefill(args, wl, W, A, Bm, ap, dev, synth, kvq, configs, torch)
        if args.phase == "merge":
            return bench_merge(args, wl, W, A, Bm, kvq, torch)
        if args.phase == "append":
            return bench_append(args, wl, dev, synth, kvq, configs, torch)
        if args.phase == "project_append":
            return bench_project_append(args, wl, W, A, Bm, ap, dev, synth, kvq, configs, torch)
        if args.phase == "prefill_attn":
            cache = fill_cache(wl, W, A, Bm, alloc_proj, dev, synth, kvq, torch, wl.context)
            return bench_prefill_attn(args, wl, cache, 1.0 / float(np.sqrt(wl.D)), dev, synth, torch)

    flush_buf = torch.empty(FLUSH_BYTES, dtype=torch.uint8, device=dev)
    copy_gbs = measure_copy(flush_buf, torch)
    steps = args.steps if args.steps is not None else wl.decode_steps
    res, state = decode_run(wl, steps, args.warmup, not args.no_warm, flush_buf, args, dev, alloc_proj, bf16,
                            np, torch, configs, kvq, synth)
    att = res["attention"]
    print(f"bench: {wl.name} done: {res['tokens_per_s']:.0f} tokens/s, attention {att['us']:.1f} us "
          f"({att['gbs']:.0f} GB/s)", file=sys.stderr, flush=True)
    traffic = measured_traffic(wl.name)
    result = {
        "metric": METRIC,
        "value": res["tokens_per_s"],
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": steps,
        "warmup": args.warmup,
        "ms_per_step": res["ms_per_step"],
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "u%d/f16" % wl.fmt["k_bits"],
        "data": "synthetic",
        "config": {"workload": wl.name, "B": wl.B, "H_q": wl.H_q, "H_kv": wl.H_kv, "head_dim": wl.D,
                   "d_in": wl.d_in, "rank": wl.rank, "context": wl.context, "decode_steps": wl.decode_steps,
                   "format": wl.fmt, "parallelism": "single-gpu"},
        "roofline": {"bound": "hbm", "kernel": "decode attention (split + merge), cold",
                     "achieved": att["gbs"], "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": att["gbs"] / HBM_PEAK_GBS, "traffic": traffic,
                     "bytes_per_launch": att["bytes_per_launch"], "us_per_launch": att["us"],
                     "us_per_launch_marker_events": att["us_marker_events"],
                     "copy_gbs": copy_gbs, "frac_of_copy": att["gbs"] / copy_gbs},
        "attention_us_per_step": att["us"],
        "projection": res["projection"],
        "append_us_per_step": res["append_us"],
        "warm": res.get("warm"),
    }
    image = None
    if not args.no_cpu_baseline:
        image = state["snapshot"].cpu().numpy()
    del state
    torch.cuda.empty_cache()
    if not args.no_per_config:
        per = {wl.name: summary(res)}
        for name in configs.WORKLOAD_ORDER:
            if name == args.workload:
                continue
            w2 = with_variants(configs.WORKLOADS[name], args)
            r2, st2 = decode_run(w2, min(PER_CONFIG_STEPS, w2.decode_steps), 3, not args.no_warm, flush_buf, args,
                                 dev, alloc_proj, bf16, np, torch, configs, kvq, synth)
            per[w2.name] = summary(r2)
            print(f"bench: {w2.name} done: attention {r2['attention']['us']:.1f} us "
                  f"({r2['attention']['gbs']:.0f} GB/s)", file=sys.stderr, flush=True)
            del st2
            torch.cuda.empty_cache()
        result["per_config"] = per
    if image is not None:
        result["cpu_baseline"] = cpu_baseline(wl, image, args, np, synth)
        print(f"bench: cpu baseline done", file=sys.stderr, flush=True)
    print(json.dumps(result))


def summary(res):
    a, p = res["attention"], res["projection"]
    out = {"tokens_per_s": res["tokens_per_s"], "ms_per_step": res["ms_per_step"],
           "attention_us": a["us"], "attention_gbs": a["gbs"], "attention_frac": a["gbs"] / HBM_PEAK_GBS,
           "attention_bytes": a["bytes_per_launch"],
           "projection_us": p["us"], "projection_gbs": p["gbs"], "projection_frac": p["gbs"] / HBM_PEAK_GBS,
           "fused_append": p["fused_append"], "append_us": res["append_us"],
           "attention_us_marker_events": a["us_marker_events"], "projection_us_marker_events": p["us_marker_events"]}
    if res.get("warm"):
        w = res["warm"]
        out.update({"warm_tokens_per_s": w["tokens_per_s"], "warm_attention_us": w["attention_us"],
                    "warm_attention_gbs": w["attention_gbs"]})
    return out


def measure_copy(buf, torch):
    """Device-to-device copy bandwidth (read + write bytes over time) of one
    half of the flush buffer into the other: the K8 reference for what a
    streaming kernel reaches on this device."""
    half = buf.numel() // 2
    src, dst = buf[:half], buf[half:]
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    reps = 10
    for _ in range(reps):
        dst.copy_(src)
    e1.record()
    torch.cuda.synchronize()
    return 2.0 * half * reps / (e0.elapsed_time(e1) * 1e-3) / 1e9


def fill_cache(wl, W, A, Bm, alloc_proj, dev, synth, kvq, torch, T_max):
    """Cache filled to the workload's context by the prefill path (projection
    of each chunk, then its append)."""
    B, Hkv, D = wl.B, wl.H_kv, wl.D
    cache = kvq.Cache(wl.fmt, B, Hkv, D, T_max, device=dev)
    chunk = min(wl.chunk, wl.context)
    Qp, Kp, Vp, wsp = alloc_proj(wl, B * chunk)
    done = 0
    while done < wl.context:
        c = min(chunk, wl.context - done)
        Hc = synth.normal_bf16_device(wl.seed, ("prefill", done), (B * c, wl.d_in), device=dev)
        kvq.project_qkv(Hc, W, A, Bm, wl.rank, wl.lora_scale, wl.d_q, wl.d_kv,
                        Qp[:B * c], Kp[:B * c], Vp[:B * c], wsp)
        cache.append(Kp[:B * c].view(B, c, Hkv, D), Vp[:B * c].view(B, c, Hkv, D))
        done += c
    torch.cuda.synchronize()
    return cache


def fused_window_step(wl) -> bool:
    """Whether a decode step can use kvq_project_append (window formats:
    the new K and V go straight into the fp16 window)."""
    f = wl.fmt
    return f["flush"] > 0 and f["rotate"] == 0 and f["sink"] == 0 and wl.B <= 32


def decode_run(wl, steps, warmup, with_warm, flush_buf, args, dev, alloc_proj, bf16, np, torch, configs, kvq,
               synth):
    """Fill the cache, then time `steps` decode steps cold (a MALL flush
    before each, outside its events) and, with `with_warm`, the same steps
    back to back.  The step timings carry events only at step boundaries;
    a second cold pass with events between the calls gives the breakdown.
    Returns (results, objects to keep alive)."""
    B, Hq, Hkv, D = wl.B, wl.H_q, wl.H_kv, wl.D
    W, A, Bm = (bf16(x) for x in synth.layer_weights(wl))
    cache = fill_cache(wl, W, A, Bm, alloc_proj, dev, synth, kvq, torch, wl.context + wl.decode_steps)
    snapshot = cache.storage.clone()
    Hdec = synth.normal_bf16_device(wl.seed, "decode", (wl.decode_steps, B, wl.d_in), device=dev)
    Qd, Kd, Vd, wsd = alloc_proj(wl, B)
    O = torch.empty((B, Hq, D), dtype=torch.float32, device=dev)
    wsa = cache.decode_workspace(Hq, device=dev)
    sm = 1.0 / float(np.sqrt(D))
    Kv, Vv, Qv = Kd.view(B, 1, Hkv, D), Vd.view(B, 1, Hkv, D), Qd.view(B, Hq, D)
    Hsteps = [Hdec[i] for i in range(wl.decode_steps)]
    fused = fused_window_step(wl)
    flush_val = [0]

    def flush():
        flush_val[0] = (flush_val[0] + 1) & 0xFF
        flush_buf.fill_(flush_val[0])

    def restart():
        # outside any timed region: the storage as it was at the context length
        cache.storage.copy_(snapshot)
        cache.restore(wl.context)

    def new_events(k):
        return [FenceFreeEvent(torch) for _ in range(k)]

    def step(i, ev=None, dev=None):
        """One decode step; ev = 4 events: before, after the projection (and
        the fused append), after the append, after the attention.  dev = 4
        events recorded by the kernels' own dispatches (kvq_time_launches):
        the projection call's first kernel start and last kernel end, then
        the attention call's."""
        if ev is not None:
            ev[0].record()
        if dev is not None:
            kvq.time_launches(dev[0].handle, dev[1].handle)
        if fused:
            kvq.project_append(Hsteps[i], W, A, Bm, wl.rank, wl.lora_scale, wl.d_q, wl.d_kv, Qd, cache, 1, wsd)
            if dev is not None:
                kvq.time_launches(None, None)
            if ev is not None:
                ev[1].record()
                ev[2].record()
        else:
            kvq.project_qkv(Hsteps[i], W, A, Bm, wl.rank, wl.lora_scale, wl.d_q, wl.d_kv, Qd, Kd, Vd, wsd)
            if dev is not None:
                kvq.time_launches(None, None)
            if ev is not None:
                ev[1].record()
            cache.append(Kv, Vv)
            if ev is not None:
                ev[2].record()
        if dev is not None:
            kvq.time_launches(dev[2].handle, dev[3].handle)
        cache.decode_attn(Qv, Hq, sm, O, wsa)
        if dev is not None:
            kvq.time_launches(None, None)
        if ev is not None:
            ev[3].record()

    if args.copy_probe_mb:
        # one elementwise kernel that reads and writes exactly this many bytes
        src = torch.empty(args.copy_probe_mb << 20, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        torch.add(src, 1, out=dst)
        torch.cuda.synchronize()
        del src, dst

    # warmup: flushed like the cold steps
    for i in range(warmup):
        if i % wl.decode_steps == 0:
            restart()
        flush()
        step(i % wl.decode_steps)
    torch.cuda.synchronize()

    def cold(breakdown):
        """The timed steps, a flush before each outside its events."""
        restart()
        n_at, evs = [], []
        torch.cuda.synchronize()
        for i in range(steps):
            j = i % wl.decode_steps
            if j == 0 and i:
                restart()
            flush()
            n_at.append(wl.context + j + 1)
            if breakdown == "dispatch":
                evs.append(new_events(4))
                step(j, dev=evs[-1])
            elif breakdown:
                evs.append(new_events(4))
                step(j, evs[-1])
            else:
                e = new_events(2)
                e[0].record()
                step(j)
                e[1].record()
                evs.append(e)
        torch.cuda.synchronize()
        return n_at, evs

    n_at, evs = cold(False)
    step_ms = np.array([e[0].elapsed_time(e[1]) for e in evs])
    _, bev = cold(True)
    proj_mk = np.array([e[0].elapsed_time(e[1]) for e in bev])
    app_ms = np.array([e[1].elapsed_time(e[2]) for e in bev])
    attn_mk = np.array([e[2].elapsed_time(e[3]) for e in bev])
    # the calls' device time from their kernels' own dispatch timestamps
    _, dev = cold("dispatch")
    proj_ms = np.array([e[0].elapsed_time(e[1]) for e in dev])
    attn_ms = np.array([e[2].elapsed_time(e[3]) for e in dev])
    bytes_launch = np.array([configs.attention_bytes(wl, n) for n in n_at], dtype=np.float64)
    proj_bytes = configs.projection_weight_bytes(wl.d_in, wl.d_q, wl.d_kv, wl.rank) + 2 * B * (wl.d_in + wl.d_qkv)
    res = {
        "tokens_per_s": B * steps / (step_ms.sum() * 1e-3),
        "ms_per_step": float(step_ms.mean()),
        "attention": {"us": float(attn_ms.mean() * 1e3), "bytes_per_launch": float(bytes_launch.mean()),
                      "gbs": float(bytes_launch.mean() / (attn_ms.mean() * 1e-3) / 1e9),
                      "us_marker_events": float(attn_mk.mean() * 1e3)},
        "projection": {"us": float(proj_ms.mean() * 1e3), "bytes_per_call": int(proj_bytes),
                       "gbs": float(proj_bytes / (proj_ms.mean() * 1e-3) / 1e9),
                       "frac": float(proj_bytes / (proj_ms.mean() * 1e-3) / 1e9 / HBM_PEAK_GBS),
                       "us_marker_events": float(proj_mk.mean() * 1e3),
                       "fused_append": fused},
        "append_us": float(app_ms.mean() * 1e3),
    }
    if with_warm:
        # the same steps back to back (at most one pass over the decode
        # inputs: the fp16 window cannot be restored inside the loop)
        done = min(steps, wl.decode_steps)
        restart()
        torch.cuda.synchronize()
        t0, t1 = new_events(2)
        t0.record()
        for i in range(done):
            step(i)
        t1.record()
        torch.cuda.synchronize()
        warm_ms = t0.elapsed_time(t1) / done
        restart()
        wev = [new_events(4) for _ in range(done)]
        torch.cuda.synchronize()
        for i in range(done):
            step(i, wev[i])
        torch.cuda.synchronize()
        wa = np.array([e[2].elapsed_time(e[3]) for e in wev])
        res["warm"] = {"tokens_per_s": B / (warm_ms * 1e-3), "ms_per_step": warm_ms, "steps": done,
                       "attention_us": float(wa.mean() * 1e3),
                       "attention_gbs": float(bytes_launch[:done].mean() / (wa.mean() * 1e-3) / 1e9)}
    restart()
    torch.cuda.synchronize()
    state = {"cache": cache, "snapshot": snapshot, "weights": (W, A, Bm), "inputs": Hdec, "workspace": wsa}
    return res, state


def cpu_baseline(wl, image, args, np, synth):
    """The oracle (C, OpenMP over independent units) on a bounded sample of
    the same workload: starting from the GPU-filled cache image at the
    context length, decode steps (projection of the B new tokens, append,
    fp64 attention over all cached tokens), timed end to end on every core
    this process may use, then one step on one thread."""
    import oracle

    cores = len(os.sched_getaffinity(0))
    model = "unknown"
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    W, A, Bm = synth.layer_weights(wl)
    ref = oracle.Cache(wl.fmt, wl.B, wl.H_kv, wl.D, wl.T_max)
    ref.image[:] = image
    ref.n = wl.context

    def one(i):
        H = synth.hidden(wl, ("cpu-sample", i), wl.B)
        _, yb = oracle.project(H, W, A, Bm, wl.rank, wl.lora_scale, wl.d_q, wl.d_kv)
        q = yb[:, :wl.d_q].reshape(wl.B, wl.H_q, wl.D)
        k = yb[:, wl.d_q:wl.d_q + wl.d_kv].reshape(wl.B, 1, wl.H_kv, wl.D)
        v = yb[:, wl.d_q + wl.d_kv:].reshape(wl.B, 1, wl.H_kv, wl.D)
        ref.append(k, v)
        ref.decode_attn(q, 1.0 / np.sqrt(wl.D))

    before = oracle.get_threads()
    try:
        oracle.set_threads(cores)
        t = time.perf_counter()
        one(0)
        first = time.perf_counter() - t
        S = int(min(max(args.cpu_seconds / max(first, 1e-3), 2), wl.decode_steps - 2))
        t = time.perf_counter()
        for i in range(1, S + 1):
            one(i)
        el = time.perf_counter() - t
        oracle.set_threads(1)
        t = time.perf_counter()
        one(S + 1)
        el1 = time.perf_counter() - t
    finally:
        oracle.set_threads(before)
    return {"value": wl.B * S / el, "unit": "tokens/s", "cores": cores, "kind": "oracle",
            "cpu_model": model, "value_1thread": wl.B / el1,
            "sample": f"{S} decode steps of {wl.name} (B={wl.B}, from context {wl.context}) on {cores} threads "
                      f"({el:.1f} s), then 1 step on 1 thread ({el1:.1f} s): oracle projection (fp64), append "
                      f"and fp64 attention over all cached tokens"}


def bench_prefill(args, wl, W, A, Bm, alloc_proj, dev, synth, kvq, configs, torch):
    """Projection GEMM at the prefill chunk (M = B * chunk rows): MFMA roofline."""
    M = wl.B * wl.chunk
    Q, K, V, ws = alloc_proj(M)
    H = synth.normal_bf16_device(wl.seed, "prefill-bench", (M, wl.d_in), device=dev)
    for _ in range(args.warmup):
        kvq.project_qkv(H, W, A, Bm, wl.rank, wl.lora_scale, wl.d_q, wl.d_kv, Q, K, V, ws)
    steps = args.steps or 20
    torch.cuda.synchronize()
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    t0.record()
    for _ in range(steps):
        kvq.project_qkv(H, W, A, Bm, wl.rank, wl.lora_scale, wl.d_q, wl.d_kv, Q, K, V, ws)
    t1.record()
    torch.cuda.synchronize()
    ms = t0.elapsed_time(t1) / steps
    flops = configs.projection_flops(M, wl.d_in, wl.d_q, wl.d_kv, wl.rank)
    tflops = flops / (ms * 1e-3) / 1e12
    print(json.dumps({
        "metric": "adapted QKV projection (prefill chunk) TFLOP/s", "value": tflops, "unit": "TFLOP/s",
        "n_gpus": 1, "steps": steps, "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": wl.name, "M": M, "d_in": wl.d_in, "d_qkv": wl.d_qkv, "rank": wl.rank},
        "roofline": {"bound": "mfma", "achieved": tflops, "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                     "frac": tflops / BF16_PEAK_TFLOPS, "traffic": None},
    }))


def bench_project_append(args, wl, W, A, Bm, alloc_proj, dev, synth, kvq, configs, torch):
    """One prefill chunk projected and appended, fused (kvq_project_append)
    against the two calls it replaces (project_qkv, then append of its bf16
    K and V): MFMA roofline on the projection's flops."""
    B, n = wl.B, wl.chunk
    M = B * n
    Q, K, V, ws = alloc_proj(M)
    H = synth.normal_bf16_device(wl.seed, "prefill-bench", (M, wl.d_in), device=dev)
    cache = kvq.Cache(wl.fmt, B, wl.H_kv, wl.D, n, device=dev)
    steps = args.steps or 20

    def fused():
        cache.reset()
        kvq.project_append(H, W, A, Bm, wl.rank, wl.lora_scale, wl.d_q, wl.d_kv, Q, cache, n, ws)

    def unfused():
        cache.reset()
        kvq.project_qkv(H, W, A, Bm, wl.rank, wl.lora_scale, wl.d_q, wl.d_kv, Q, K, V, ws)
        cache.append(K.view(B, n, wl.H_kv, wl.D), V.view(B, n, wl.H_kv, wl.D))

    def timed(fn):
        for _ in range(args.warmup):
            fn()
        torch.cuda.synchronize()
        t0 = torch.cuda.Event(enable_timing=True)
        t1 = torch.cuda.Event(enable_timing=True)
        t0.record()
        for _ in range(steps):
            fn()
        t1.record()
        torch.cuda.synchronize()
        return t0.elapsed_time(t1) / steps

    ms_unfused = timed(unfused)
    ms = timed(fused)
    flops = configs.projection_flops(M, wl.d_in, wl.d_q, wl.d_kv, wl.rank)
    tflops = flops / (ms * 1e-3) / 1e12
    print(json.dumps({
        "metric": "fused projection + append (prefill chunk) TFLOP/s", "value": tflops, "unit": "TFLOP/s",
        "n_gpus": 1, "steps": steps, "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": wl.name, "M": M, "d_in": wl.d_in, "d_qkv": wl.d_qkv, "rank": wl.rank},
        "unfused_ms_per_step": ms_unfused,
        "roofline": {"bound": "mfma", "achieved": tflops, "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                     "frac": tflops / BF16_PEAK_TFLOPS, "traffic": None},
    }))


def bench_prefill_attn(args, wl, cache, sm, dev, synth, torch):
    """Causal attention of the last prefill chunk (C = the workload's chunk,
    its tokens already appended) over the packed cache of `context` tokens.
    Algorithmic flops: 4 D per (query head, visible key), i.e.
    4 B H_q D (C (n - C) + C (C + 1) / 2), against the dense fp16 MFMA peak."""
    B, Hq, D = wl.B, wl.H_q, wl.D
    C, n = wl.chunk, wl.context
    Q = synth.normal_bf16_device(wl.seed, "prefill-attn-q", (B, C, Hq, D), device=dev)
    O = torch.empty((B, C, Hq, D), dtype=torch.float32, device=dev)
    ws = cache.prefill_workspace(dev)
    for _ in range(args.warmup):
        cache.prefill_attn(Q, C, Hq, sm, O, ws)
    steps = args.steps or 20
    torch.cuda.synchronize()
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    t0.record()
    for _ in range(steps):
        cache.prefill_attn(Q, C, Hq, sm, O, ws)
    t1.record()
    torch.cuda.synchronize()
    ms = t0.elapsed_time(t1) / steps
    flops = 4.0 * B * Hq * D * (C * (n - C) + C * (C + 1) / 2)
    tflops = flops / (ms * 1e-3) / 1e12
    print(json.dumps({
        "metric": "chunked prefill attention TFLOP/s", "value": tflops, "unit": "TFLOP/s",
        "n_gpus": 1, "steps": steps, "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "u%d/f16" % wl.fmt["k_bits"], "data": "synthetic",
        "config": {"workload": wl.name, "B": B, "H_q": Hq, "H_kv": wl.H_kv, "head_dim": D, "chunk": C,
                   "context": n, "format": wl.fmt},
        "roofline": {"bound": "mfma", "achieved": tflops, "peak": BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                     "frac": tflops / BF16_PEAK_TFLOPS, "traffic": None},
    }))


def bench_merge(args, wl, W, A, Bm, kvq, torch):
    """Dense adapter merge W' = W + s B_p A_p (Sec. 3.4 deployment): HBM roofline.
    Algorithmic bytes: read W, A, B and write W' once, all bf16."""
    out = torch.empty_like(W)
    for _ in range(args.warmup):
        kvq.merge_adapter(W, A, Bm, wl.rank, wl.lora_scale, wl.d_q, wl.d_kv, out)
    steps = args.steps or 50
    torch.cuda.synchronize()
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    t0.record()
    for _ in range(steps):
        kvq.merge_adapter(W, A, Bm, wl.rank, wl.lora_scale, wl.d_q, wl.d_kv, out)
    t1.record()
    torch.cuda.synchronize()
    ms = t0.elapsed_time(t1) / steps
    nbytes = 2 * (2 * W.numel() + A.numel() + Bm.numel())
    gbs = nbytes / (ms * 1e-3) / 1e9
    print(json.dumps({
        "metric": "dense adapter merge GB/s", "value": gbs, "unit": "GB/s",
        "n_gpus": 1, "steps": steps, "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": wl.name, "d_in": wl.d_in, "d_qkv": wl.d_qkv, "rank": wl.rank},
        "roofline": {"bound": "hbm", "achieved": gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": gbs / HBM_PEAK_GBS, "traffic": None},
    }))


def bench_append(args, wl, dev, synth, kvq, configs, torch):
    """Quantize-and-pack append of one prefill chunk (the workload's chunk
    tokens per sequence) into an empty cache: HBM roofline.  Algorithmic
    bytes: read the bf16 K and V once; write the codes and metadata of the
    coded tokens and the fp16 rows of sink and window tokens."""
    B, H, D, n = wl.B, wl.H_kv, wl.D, wl.chunk
    K = synth.normal_bf16_device(wl.seed, "append-k", (B, n, H, D), device=dev)
    V = synth.normal_bf16_device(wl.seed, "append-v", (B, n, H, D), device=dev)
    cache = kvq.Cache(wl.fmt, B, H, D, n, device=dev)
    if args.copy_probe_mb:
        # one elementwise kernel that reads and writes exactly this many bytes
        src = torch.empty(args.copy_probe_mb << 20, dtype=torch.uint8, device=dev)
        dst = torch.empty_like(src)
        torch.add(src, 1, out=dst)
        torch.cuda.synchronize()
        del src, dst
    for _ in range(args.warmup):
        cache.reset()
        cache.append(K, V)
    steps = args.steps or 50
    torch.cuda.synchronize()
    t0 = torch.cuda.Event(enable_timing=True)
    t1 = torch.cuda.Event(enable_timing=True)
    t0.record()
    for _ in range(steps):
        cache.reset()  # host-only: the next append rewrites every live byte
        cache.append(K, V)
    t1.record()
    torch.cuda.synchronize()
    ms = t0.elapsed_time(t1) / steps
    f = wl.fmt
    nq = configs.num_coded(f, n)
    m16 = f.get("meta_fp16", 0)
    bk = configs.coded_bytes_per_token(D, f["k_bits"], f["k_axis"], f["k_group"], f["k_mode"] == configs.AFFINE, m16)
    bv = configs.coded_bytes_per_token(D, f["v_bits"], f["v_axis"], f["v_group"], f["v_mode"] == configs.AFFINE, m16)
    nbytes = 2 * 2 * B * n * H * D + B * H * (nq * (bk + bv) + (n - nq) * 4 * D)
    gbs = nbytes / (ms * 1e-3) / 1e9
    print(json.dumps({
        "metric": "prefill-chunk append GB/s", "value": gbs, "unit": "GB/s",
        "n_gpus": 1, "steps": steps, "warmup": args.warmup, "ms_per_step": ms, "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "u%d/f16" % f["k_bits"], "data": "synthetic",
        "config": {"workload": wl.name, "B": B, "tokens": n, "H_kv": H, "head_dim": D, "format": f},
        "roofline": {"bound": "hbm", "achieved": gbs, "peak": HBM_PEAK_GBS, "unit": "GB/s",
                     "frac": gbs / HBM_PEAK_GBS, "traffic": None, "bytes_per_launch": nbytes},
    }))


if __name__ == "__main__":
    main()
