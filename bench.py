"""Benchmark of the visual-memory path on one MI355X.

A step is one pass of the whole path over one batch: the all-layer down
projection, the per-layer memories + RMSNorm + visual K/V projection for every
layer, and the text-query attention of every layer. The default workload is
the LLaVA-1.5-7B-shaped batch (4 sequences x 576 visual + 64 text tokens, 32
layers, bf16). Inputs are seeded synthetic tensors already resident in HBM when
the timed region starts.

Prints one JSON line with the whole-step throughput, a roofline entry for the
dominant kernel (timed with HIP events around its own launches inside the timed
region), per-stage figures and a CPU baseline of the fp64 oracle.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "visual tokens/sec (memory build+KV) & text-attn TFLOP/s; % MFMA / HBM peak"
PEAK_BF16_TFLOPS = 2516.6   # 256 CU x 2.4 GHz x 4096 dense bf16 FLOP/clk/CU
PEAK_F32_TFLOPS = 157.3
PEAK_HBM_GBS = 8000.0


def log(*a):
    print(*a, file=sys.stderr, flush=True)


class HipEvents:
    """Raw hipEvent_t handles from the HIP runtime (the library records them itself)."""

    def __init__(self):
        import ctypes
        self.ct = ctypes
        self.hip = ctypes.CDLL("libamdhip64.so")
        self.hip.hipEventCreate.argtypes = [ctypes.POINTER(ctypes.c_void_p)]
        self.hip.hipEventElapsedTime.argtypes = [ctypes.POINTER(ctypes.c_float), ctypes.c_void_p,
                                                 ctypes.c_void_p]
        self.hip.hipEventDestroy.argtypes = [ctypes.c_void_p]
        self.made = []

    def new(self) -> int:
        h = self.ct.c_void_p()
        if self.hip.hipEventCreate(self.ct.byref(h)) != 0:
            raise RuntimeError("hipEventCreate failed")
        self.made.append(h.value)
        return h.value

    def pair(self):
        return self.new(), self.new()

    def ms(self, pair) -> float:
        out = self.ct.c_float()
        rc = self.hip.hipEventElapsedTime(self.ct.byref(out), pair[0], pair[1])
        if rc != 0:
            raise RuntimeError(f"hipEventElapsedTime failed ({rc})")
        return float(out.value)

    def close(self):
        for h in self.made:
            self.hip.hipEventDestroy(h)
        self.made = []


def parse():
    p = argparse.ArgumentParser()
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=20)
    p.add_argument("--warmup", type=int, default=5)
    p.add_argument("--workload", default="llava7b",
                   choices=["llava7b", "llava_next", "qwen25vl_video", "decode", "tiny",
                            "gdn_video", "gdn_image"])
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--no-decode", action="store_true",
                   help="skip the decode-shape measurement appended to prefill workloads")
    p.add_argument("--no-cold", action="store_true",
                   help="skip the cold-cache steps (512 MiB rewritten before each)")
    p.add_argument("--no-workloads", action="store_true",
                   help="skip the compact LLaVA-NeXT and Qwen2.5-VL video blocks appended to the "
                        "default LLaVA-7B run")
    p.add_argument("--no-delta", action="store_true",
                   help="skip the linear-attention visual write appended to prefill workloads")
    p.add_argument("--no-variants", action="store_true",
                   help="skip the recurrent-adapter and layer-skipping measurements")
    p.add_argument("--calibrate-copy", action="store_true",
                   help="also run a plain 1 GiB device copy, whose memory counters calibrate the "
                        "FETCH_SIZE / WRITE_SIZE readings of the kernels")
    return p.parse_args()


# Sources of the dominant kernel: a stored counter measurement is only used while they match.
KV_SOURCES = ("paper_2609_34972_amd/csrc/gemm_pipe.hpp", "paper_2609_34972_amd/csrc/build_kernels.hip",
              "paper_2609_34972_amd/csrc/dv_device.hpp")
TRAFFIC_FILE = "profiles/k_kv_proj_llava7b_traffic.txt"


def sources_digest(paths=KV_SOURCES) -> str:
    import hashlib
    h = hashlib.sha256()
    for p in paths:
        with open(os.path.join(ROOT, p), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


ATTN_SOURCES = ("paper_2609_34972_amd/csrc/attention.hip", "paper_2609_34972_amd/csrc/attention.hpp",
                "paper_2609_34972_amd/csrc/gemm_pipe.hpp", "paper_2609_34972_amd/csrc/dv_device.hpp")
DECODE_TRAFFIC_FILE = "profiles/k_attn_decode_traffic.txt"


def stored_counters(path=TRAFFIC_FILE, sources=KV_SOURCES):
    """Key/value lines of a committed counter summary, or None once the kernel's sources have
    changed since the counters were taken."""
    path = os.path.join(ROOT, path)
    if not os.path.exists(path):
        return None
    kv = {}
    for line in open(path):
        if ":" in line and not line.startswith("#"):
            k, v = line.split(":", 1)
            kv[k.strip()] = v.strip()
    if kv.get("sources_sha256_16") != sources_digest(sources):
        return None
    return kv


def stored_traffic(path=TRAFFIC_FILE, sources=KV_SOURCES):
    """HBM bytes per launch from the committed counter summary, if still current."""
    kv = stored_counters(path, sources)
    try:
        return float(kv["traffic_bytes_per_launch"]) if kv else None
    except (KeyError, ValueError):
        return None


def cpu_model() -> str:
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    import platform
    return platform.processor() or "unknown"


def provenance():
    """Which sources produced the numbers: the git revision the library was built at (recorded
    by the build, since runs may happen where no git metadata exists), whether that tree had
    uncommitted changes, and a digest of the library sources as they are now."""
    from paper_2609_34972_amd import build as hip_build
    info = {}
    try:
        with open(hip_build.INFO) as f:
            info = json.load(f)
    except (OSError, ValueError):
        pass
    now = hip_build.sources_digest()
    return {"git_rev": info.get("git_rev"), "git_dirty_at_build": info.get("git_dirty"),
            "sources_sha256_16": now,
            "library_built_from_these_sources": info.get("sources_sha256_16") == now,
            "cpu_model": cpu_model(), "host_threads": os.cpu_count()}


def percentiles(xs):
    import numpy as np
    a = np.asarray(xs, dtype=np.float64)
    return {"median": float(np.median(a)), "p10": float(np.percentile(a, 10)),
            "p90": float(np.percentile(a, 90))}


def time_calls(fn, steps, warmup, flush=None):
    """Per-call times (ms) of fn() from torch events on the current stream. With flush, a
    buffer larger than the last-level cache is rewritten before every call, outside the
    timed events (cold runs)."""
    import torch
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    mk = lambda: torch.cuda.Event(enable_timing=True)
    pairs = [(mk(), mk()) for _ in range(steps)]
    for a, b in pairs:
        if flush is not None:
            flush.add_(1)
        a.record()
        fn()
        b.record()
    torch.cuda.synchronize()
    return [a.elapsed_time(b) for a, b in pairs]


def cpu_baseline(w, E, wts, tx, vcache):
    """Time the fp64 oracle on a bounded sample of the same workload and scale it to the step."""
    import numpy as np
    import torch

    import oracle
    from paper_2609_34972_amd import configs, synth

    f64 = synth.as_f64
    threads = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))
    tok, nl = min(2048, w.T), min(8, w.L)
    E64 = f64(E[:tok])
    li = torch.arange(nl)
    Dw, Uw, g = f64(wts["Dw"][li]), f64(wts["Uw"][li]), f64(wts["gamma"][li])
    Wk, Wv = f64(wts["Wk"][li]), f64(wts["Wv"][li])
    t0 = time.perf_counter()
    Z = oracle.down(E64, Dw, w.act)
    oracle.project_visual_kv(E64, Z, Uw, g, Wk, Wv, 1, tok, w.Hkv, w.hd, w.eps)
    t_build = time.perf_counter() - t0
    build_per_token = t_build / tok * (w.L / nl)
    groups = min(32, w.B * w.Hkv)
    t0 = time.perf_counter()
    for k in range(groups):
        b, g = k % w.B, (k // w.B) % w.Hkv
        hs = slice(g * w.G, (g + 1) * w.G)
        oracle.text_visual_attention(f64(tx["Q"][0][b:b + 1, :, hs]),
                                     f64(vcache["Kv"][0][b:b + 1, g:g + 1]),
                                     f64(vcache["Vv"][0][b:b + 1, g:g + 1]),
                                     f64(tx["Kt"][0][b:b + 1, g:g + 1]),
                                     f64(tx["Vt"][0][b:b + 1, g:g + 1]), w.q_pos0)
    t_attn = (time.perf_counter() - t0) / groups * (w.B * w.Hkv) * w.L
    t_step = build_per_token * w.T + t_attn
    f_build = w.T / tok * w.L / nl
    f_attn = w.B * w.Hkv * w.L / groups
    return {
        "value": w.T / t_step,
        "unit": "visual tokens/s",
        "cores": threads,
        "kind": "oracle",
        "cpu_model": cpu_model(),
        "scale_build": f_build,
        "scale_attention": f_attn,
        "sample": (f"fp64 oracle: build+KV of {tok} tokens x {nl} of {w.L} layers "
                   f"({t_build:.2f} s, scaled x{f_build:.4g}); attention of "
                   f"{groups} (batch, kv-head) groups of one layer ({t_attn / f_attn:.2f} s, "
                   f"scaled x{f_attn:.4g}); whole step {t_step:.1f} s"),
    }


def mfma_probe(iters=2048, reps=3):
    """Sustained bf16 MFMA rate of this GPU on register operands (no memory traffic), on random
    and on constant operands: the clock, and so the rate, depends on how much the operands toggle.
    Runs outside every timed region."""
    import torch

    import paper_2609_34972_amd as dvl
    sink = torch.empty(dvl.PROBE_BLOCKS, dtype=torch.float32, device="cuda:0")
    out = {"iters": iters}
    for name, rnd in (("random_bf16_tflops", True), ("constant_tflops", False)):
        dvl.probe_mfma(rnd, 256, sink)
        ts = []
        for _ in range(reps):
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record()
            dvl.probe_mfma(rnd, iters, sink)
            b.record()
            torch.cuda.synchronize()
            ts.append(a.elapsed_time(b))
        ts.sort()
        out[name] = dvl.PROBE_FLOP_PER_ITER * iters / (ts[len(ts) // 2] * 1e-3) / 1e12
    return out


def alloc_step(w, Eg, tg):
    """Outputs and workspaces of one step (all layers projected in one call)."""
    import torch

    import paper_2609_34972_amd as dvl

    dev, dt = Eg.device, Eg.dtype
    buf = {
        "Z": torch.empty(w.L, w.T, w.r, dtype=dt, device=dev),
        "Kv": torch.empty(w.L, w.B, w.Hkv, w.Nv, w.hd, dtype=dt, device=dev),
        "O": torch.empty_like(tg["Q"]),
        "ws_kv": torch.empty(dvl.project_visual_kv_workspace(w.T, w.d, w.L, dt), dtype=torch.uint8,
                             device=dev),
    }
    buf["Vv"] = torch.empty_like(buf["Kv"])
    na = dvl.text_visual_attention_workspace(w.B, w.Hq, w.Hkv, w.hd, w.Nv, w.Nq, w.Nkt)
    buf["ws_at"] = torch.empty(max(na, 16), dtype=torch.uint8, device=dev)
    return buf


def make_step(w, Eg, wg, tg, buf):
    """One pass of the whole path: the all-layer down projection, the memories + norm + K/V of
    every layer, and the attention of every layer. `ev` brackets the three build launches with
    HIP events; `attn_span`, a pair of events on torch's current stream (the library's stream
    here), brackets the attention launches of all layers, which then run back to back as in a
    timed step."""
    import paper_2609_34972_amd as dvl

    Z, Kv, Vv, O = buf["Z"], buf["Kv"], buf["Vv"], buf["O"]

    def step(ev=None, attn_span=None):
        if ev is not None:
            dvl.time_kernel(dvl.KERNEL_DOWN, *ev["down"])
            dvl.time_kernel(dvl.KERNEL_UP, *ev["up"])
            dvl.time_kernel(dvl.KERNEL_KV, *ev["kv"])
        dvl.build_visual_memory(Eg, wg["Dw"], Z, act=w.act)
        dvl.project_visual_kv(Eg, Z, wg["Uw"], wg["gamma"], wg["Wk"], wg["Wv"], Kv, Vv, eps=w.eps,
                              ws=buf["ws_kv"])
        if ev is not None:
            for k in (dvl.KERNEL_DOWN, dvl.KERNEL_UP, dvl.KERNEL_KV):
                dvl.time_kernel(k)
        if attn_span is not None:
            attn_span[0].record()
        for l in range(w.L):
            dvl.text_visual_attention(tg["Q"][l], Kv[l], Vv[l], tg["Kt"][l], tg["Vt"][l], O[l],
                                      q_pos0=w.q_pos0, ws=buf["ws_at"])
        if attn_span is not None:
            attn_span[1].record()

    return step


def fused_path(w) -> bool:
    """Whether this workload's projection takes the fused up + norm + K/V kernel (then the K/V
    events bracket that kernel and the up-projection events record nothing)."""
    import torch

    import paper_2609_34972_amd as dvl
    dt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    return dvl.project_visual_kv_fused(w.d, w.r, w.Hkv, w.hd, dt)


def measure_step(w, step, steps, warmup, n_attn_steps=3):
    """Time `steps` whole steps (the three build launches bracketed by HIP events inside the
    timed region), then time the attention launches of every layer in `n_attn_steps` extra steps,
    back to back between one pair of events (an event pair around each short launch would add
    its dispatch latency to every launch)."""
    import torch

    fused = fused_path(w)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    hev = HipEvents()
    evs = [{"down": hev.pair(), "up": hev.pair(), "kv": hev.pair()} for _ in range(steps)]
    mk = lambda: torch.cuda.Event(enable_timing=True)
    attn_spans = [(mk(), mk()) for _ in range(n_attn_steps)]
    t_begin, t_end = mk(), mk()
    marks = [mk() for _ in range(steps + 1)]
    torch.cuda.synchronize()
    t_begin.record()
    for s in range(steps):
        marks[s].record()
        step(evs[s])
    marks[-1].record()
    t_end.record()
    torch.cuda.synchronize()
    step_ms = [marks[i].elapsed_time(marks[i + 1]) for i in range(steps)]
    for s in range(n_attn_steps):
        step(attn_span=attn_spans[s])
    torch.cuda.synchronize()
    avg = lambda key: sum(hev.ms(e[key]) for e in evs) / steps
    m = {"ms_step": t_begin.elapsed_time(t_end) / steps, "step_ms": step_ms, "fused": fused,
         "down": avg("down"), "up": 0.0 if fused else avg("up"), "kv": avg("kv"),
         "attn_launch": sum(b.elapsed_time(e) for b, e in attn_spans) / (n_attn_steps * w.L)}
    hev.close()
    return m


def step_figures(w, m, peak):
    """Per-stage rates of a measured step against their bounds."""
    from paper_2609_34972_amd import configs

    f_down = 2.0 * w.T * w.d * w.r * w.L
    f_up = 2.0 * w.T * w.r * w.d * w.L
    f_kv = 2.0 * w.T * 2 * w.kv * w.d * w.L
    f_build = f_down + f_up + f_kv
    f_attn = configs.flops_attention(w)
    b_attn = configs.bytes_attention(w)
    ms_build = m["down"] + m["up"] + m["kv"]
    ms_attn_total = m["ms_step"] - ms_build
    ms_al = m["attn_launch"]
    fused = m.get("fused", False)
    # the fused kernel does the up-projection's work too
    f_kv_kernel = f_kv + f_up if fused else f_kv
    return {
        "f_kv": f_kv_kernel, "f_build": f_build, "f_attn": f_attn, "fused": fused,
        "kv_kernel": "k_up_kv_fused" if fused else "k_kv_proj",
        "kv_tflops": f_kv_kernel / (m["kv"] * 1e-3) / 1e12,
        "stages": {
            "build_kv_visual_tokens_per_s": w.T / (ms_build * 1e-3),
            "build_kv_ms": ms_build,
            "build_kv_tflops": f_build / (ms_build * 1e-3) / 1e12,
            "build_kv_mfma_frac": f_build / (ms_build * 1e-3) / 1e12 / peak,
            "down_ms": m["down"], "up_ms": m["up"], "kv_ms": m["kv"],
            "down_mfma_frac": f_down / (m["down"] * 1e-3) / 1e12 / peak,
            "up_mfma_frac": None if fused else f_up / (m["up"] * 1e-3) / 1e12 / peak,
            "kv_mfma_frac": f_kv_kernel / (m["kv"] * 1e-3) / 1e12 / peak,
            "attention_ms_all_layers": ms_attn_total,
            "attention_kernel_ms_per_layer": ms_al,
            "attention_tflops": f_attn / (ms_attn_total * 1e-3) / 1e12,
            "attention_gbs": b_attn / (ms_attn_total * 1e-3) / 1e9,
            "attention_hbm_frac": b_attn / (ms_attn_total * 1e-3) / 1e9 / PEAK_HBM_GBS,
            "attention_kernel_gbs": b_attn / w.L / (ms_al * 1e-3) / 1e9,
            "attention_kernel_hbm_frac": b_attn / w.L / (ms_al * 1e-3) / 1e9 / PEAK_HBM_GBS,
            "attention_kernel_mfma_frac": f_attn / w.L / (ms_al * 1e-3) / 1e12 / peak,
            "step_mfma_frac": (f_build + f_attn) / (m["ms_step"] * 1e-3) / 1e12 / peak,
        },
    }


def run_prefill(args, w):
    import torch

    from paper_2609_34972_amd import synth

    dev = torch.device("cuda:0")
    log(f"[bench] generating {w.name} inputs")
    E = synth.make_E(w)
    wts = synth.make_build_weights(w)
    tx = synth.make_text(w)
    Eg = E.to(dev)
    wg = {k: v.to(dev) for k, v in wts.items()}
    tg = {k: v.to(dev) for k, v in tx.items()}
    buf = alloc_step(w, Eg, tg)
    step = make_step(w, Eg, wg, tg, buf)
    log(f"[bench] warmup {args.warmup}, timing {args.steps} steps")
    m = measure_step(w, step, args.steps, args.warmup)
    peak = PEAK_BF16_TFLOPS if w.dtype == "bf16" else PEAK_F32_TFLOPS
    fig = step_figures(w, m, peak)
    ms_step, kv_tflops = m["ms_step"], fig["kv_tflops"]
    out = {
        "metric": METRIC,
        "value": w.T / (ms_step * 1e-3),
        "unit": "visual tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": w.dtype,
        "data": "synthetic",
        "config": {"workload": w.name, "batch": w.B, "visual_tokens": w.Nv, "text_tokens": w.Nt,
                   "layers": w.L, "d": w.d, "rank": w.r, "q_heads": w.Hq, "kv_heads": w.Hkv,
                   "head_dim": w.hd},
        "roofline": {"bound": "mfma", "kernel": fig["kv_kernel"], "achieved": kv_tflops, "peak": peak,
                     "unit": "TFLOP/s", "frac": kv_tflops / peak,
                     "traffic": stored_traffic() if w.name == "llava7b" else None,
                     "algorithmic_flops_per_launch": fig["f_kv"], "ms_per_launch": m["kv"]},
        "stages": fig["stages"],
    }
    out["target"] = {
        "what": "whole step (build + K/V + attention of every layer): algorithmic FLOPs / step "
                "time / bf16 MFMA peak",
        "value": fig["stages"]["step_mfma_frac"], "goal": 0.60,
        "met": fig["stages"]["step_mfma_frac"] >= 0.60,
        "step_ms_for_goal": (fig["f_build"] + fig["f_attn"]) / (0.60 * peak * 1e12) * 1e3}
    out["step_ms_warm"] = percentiles(m["step_ms"])
    if w.dtype == "bf16":
        log("[bench] MFMA-rate probe")
        probe = mfma_probe()
        probe["kernel_frac_of_random"] = kv_tflops / probe["random_bf16_tflops"]
        out["roofline"]["mfma_probe"] = probe
    if not args.no_cold:
        log("[bench] cold steps (512 MiB rewritten between steps)")
        flush = torch.empty(128 << 20, dtype=torch.float32, device=dev)
        out["step_ms_cold"] = percentiles(time_calls(step, max(3, args.steps // 4), 1, flush))
        del flush
    if not args.no_variants:
        out["variants"] = run_variants(args, w, Eg, wg, tg, peak, fig["f_build"], ms_step)
    if not args.no_cpu_baseline:
        log("[bench] timing the CPU oracle baseline")
        vc = synth.make_visual_cache(w, layers=[0])
        out["cpu_baseline"] = cpu_baseline(w, E, wts, {k: v[:1] for k, v in tx.items()}, vc)
    del Eg, wg, tg, buf, step
    torch.cuda.empty_cache()
    return out


def run_workload_block(args, w):
    """Compact figures of another prefill workload, inputs drawn on the GPU (same distributions
    as the numpy generator, which would take minutes at these sizes)."""
    import torch

    from paper_2609_34972_amd import synth

    dev = torch.device("cuda:0")
    log(f"[bench] {w.name}: generating inputs on the GPU")
    x = synth.make_on_device(w, dev, seed=0)
    Eg = x.pop("E")
    tg = {k: x.pop(k) for k in ("Q", "Kt", "Vt")}
    wg = x
    buf = alloc_step(w, Eg, tg)
    step = make_step(w, Eg, wg, tg, buf)
    steps = max(5, args.steps // 2)
    log(f"[bench] {w.name}: timing {steps} steps")
    m = measure_step(w, step, steps, 2)
    peak = PEAK_BF16_TFLOPS
    fig = step_figures(w, m, peak)
    st = fig["stages"]
    mfma_bound = w.Hq // w.Hkv * w.Nq > 315  # attention arithmetic intensity above the ridge
    res = {
        "config": {"batch": w.B, "visual_tokens": w.Nv, "text_tokens": w.Nt, "layers": w.L,
                   "d": w.d, "rank": w.r, "q_heads": w.Hq, "kv_heads": w.Hkv, "head_dim": w.hd},
        "data": "synthetic, drawn on the GPU",
        "ms_per_step": m["ms_step"], "step_ms_warm": percentiles(m["step_ms"]),
        "visual_tokens_per_s": w.T / (m["ms_step"] * 1e-3),
        "step_mfma_frac": st["step_mfma_frac"],
        "build_kv_ms": st["build_kv_ms"], "build_kv_mfma_frac": st["build_kv_mfma_frac"],
        "down_ms": st["down_ms"], "up_ms": st["up_ms"], "fused_up_kv": fig["fused"],
        "k_kv_proj": {"kernel": fig["kv_kernel"], "ms": m["kv"], "tflops": fig["kv_tflops"],
                      "frac": fig["kv_tflops"] / peak},
        "attention": {"kernel_ms_per_layer": m["attn_launch"],
                      "bound": "mfma" if mfma_bound else "hbm",
                      "frac": st["attention_kernel_mfma_frac"] if mfma_bound
                      else st["attention_kernel_hbm_frac"],
                      "tflops": fig["f_attn"] / w.L / (m["attn_launch"] * 1e-3) / 1e12,
                      "gbs": st["attention_kernel_gbs"],
                      "ms_all_layers_in_step": st["attention_ms_all_layers"]},
    }
    dt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    import paper_2609_34972_amd as dvl
    dvl.set_fused_kv(True)
    try:
        if dvl.project_visual_kv_fused(w.d, w.r, w.Hkv, w.hd, dt):
            # the fused up + norm + K/V kernel (off by default), timed on the same inputs
            log(f"[bench] {w.name}: timing the fused up + norm + K/V variant")
            mf = measure_step(w, step, max(3, steps // 2), 1, n_attn_steps=1)
            ff = step_figures(w, mf, peak)
            res["fused_up_kv_variant"] = {
                "ms_per_step": mf["ms_step"], "build_kv_ms": ff["stages"]["build_kv_ms"],
                "kernel": ff["kv_kernel"], "kernel_ms": mf["kv"], "tflops": ff["kv_tflops"],
                "frac": ff["kv_tflops"] / peak,
                "vs_default_up_plus_kv_ms": m["up"] + m["kv"]}
    finally:
        dvl.set_fused_kv(False)
    del x, Eg, tg, wg, buf, step
    torch.cuda.empty_cache()
    return res


def run_variants(args, w, Eg, wg, tg, peak, f_build, ms_full_step):
    """The recurrent adapter (Eq. 6) and layer-wise adapter skipping on the same inputs."""
    import torch

    import paper_2609_34972_amd as dvl
    from paper_2609_34972_amd import configs

    dev = Eg.device
    dt = Eg.dtype
    res = {}
    steps, warm = max(5, args.steps // 2), 2
    # recurrent adapter: per-layer chain, then the K/V projection of every layer
    log("[bench] variant: recurrent adapter")
    Kv = torch.empty(w.L, w.B, w.Hkv, w.Nv, w.hd, dtype=dt, device=dev)
    Vv = torch.empty_like(Kv)
    ws = torch.empty(dvl.recurrent_visual_kv_workspace(w.T, w.d, w.L, w.r, dt), dtype=torch.uint8,
                     device=dev)
    t = percentiles(time_calls(lambda: dvl.recurrent_visual_kv(
        Eg, wg["Dw"], wg["Uw"], wg["gamma"], wg["Wk"], wg["Wv"], Kv, Vv, eps=w.eps, act=w.act,
        ws=ws), steps, warm))
    res["recurrent_build_kv"] = {
        "ms": t, "visual_tokens_per_s": w.T / (t["median"] * 1e-3),
        "tflops": f_build / (t["median"] * 1e-3) / 1e12,
        "mfma_frac": f_build / (t["median"] * 1e-3) / 1e12 / peak}
    del Kv, Vv, ws
    # adapter skipping as in the appendix tables: first 5 and last 10 layers skipped
    if w.L > 15:
        keep = [0] * 5 + [1] * (w.L - 15) + [0] * 10
        nk = sum(keep)
        log(f"[bench] variant: adapters of the first 5 and last 10 layers skipped ({nk} kept)")
        Kv = torch.empty(nk, w.B, w.Hkv, w.Nv, w.hd, dtype=dt, device=dev)
        Vv = torch.empty_like(Kv)
        ws = torch.empty(dvl.kept_visual_kv_workspace(w.T, w.d, w.r, nk, dt), dtype=torch.uint8,
                         device=dev)
        O = torch.empty_like(tg["Q"])
        na = dvl.text_visual_attention_workspace(w.B, w.Hq, w.Hkv, w.hd, w.Nv, w.Nq, w.Nkt)
        wsa = torch.empty(max(na, 16), dtype=torch.uint8, device=dev)
        slot = {l: j for j, l in enumerate(l for l in range(w.L) if keep[l])}

        def kept_step():
            dvl.kept_visual_kv(Eg, wg["Dw"], wg["Uw"], wg["gamma"], wg["Wk"], wg["Wv"], keep, Kv,
                               Vv, eps=w.eps, act=w.act, ws=ws)
            for l in range(w.L):
                j = slot.get(l)
                dvl.text_visual_attention(tg["Q"][l], Kv[j] if j is not None else None,
                                          Vv[j] if j is not None else None, tg["Kt"][l],
                                          tg["Vt"][l], O[l], q_pos0=w.q_pos0, ws=wsa)

        t = percentiles(time_calls(kept_step, steps, warm))
        res["skip_first5_last10"] = {
            "kept_layers": nk, "ms_per_step": t,
            "visual_tokens_per_s": w.T / (t["median"] * 1e-3),
            "speedup_vs_all_layers": ms_full_step / t["median"],
            "visual_cache_bytes": 2 * Kv.numel() * Kv.element_size(),
            "visual_cache_bytes_all_layers": 2 * w.L * w.T * w.kv * Kv.element_size()}
        del Kv, Vv, ws, O, wsa
    # backbone epilogue of the visual K/V: the rotary embedding of the visual keys at their
    # positions (a multimodal 16/24/24 rotation over a 16 x 32 x 32 video grid plus the K/V
    # bias for the video workload, 1-D rotation after a 35-token prompt otherwise)
    from paper_2609_34972_amd import synth
    video = w.name == "qwen25vl_video"
    log("[bench] variant: backbone epilogue")
    Z = torch.empty(w.L, w.T, w.r, dtype=dt, device=dev)
    Kv = torch.empty(w.L, w.B, w.Hkv, w.Nv, w.hd, dtype=dt, device=dev)
    Vv = torch.empty_like(Kv)
    if video:
        ew = {k: v.to(dev) for k, v in synth.make_epilogue_weights(w).items()}
        epi = dvl.KVEpilogue(k_bias=ew["k_bias"], v_bias=ew["v_bias"],
                             positions=synth.video_positions(w.B, 16, 32, 32, 15).to(dev),
                             rope_sections=(16, 24, 24), rope_theta=1e6)
        feats = "k/v bias + multimodal rotary embedding (16/24/24, theta 1e6)"
    else:
        epi = dvl.KVEpilogue(positions=synth.image_positions(w.B, w.Nv, 35).to(dev))
        feats = "rotary embedding (theta 1e4) at positions 35..35+Nv-1"
    ws = torch.empty(dvl.project_visual_kv_ex_workspace(w.T, w.d, w.L, w.hd, dt),
                     dtype=torch.uint8, device=dev)

    def build(e):
        dvl.build_visual_memory(Eg, wg["Dw"], Z, act=w.act)
        dvl.project_visual_kv(Eg, Z, wg["Uw"], wg["gamma"], wg["Wk"], wg["Wv"], Kv, Vv, eps=w.eps,
                              ws=ws, epilogue=e)

    t_plain = percentiles(time_calls(lambda: build(None), steps, warm))
    t_epi = percentiles(time_calls(lambda: build(epi), steps, warm))
    res["backbone_epilogue"] = {
        "features": feats, "build_kv_ms": t_epi, "build_kv_ms_plain": t_plain,
        "overhead_frac": t_epi["median"] / t_plain["median"] - 1.0}
    del Z, Kv, Vv, ws, epi
    torch.cuda.empty_cache()
    return res


def run_delta(args, w, steps=None, warmup=None):
    """Visual write into the linear-attention states of a hybrid Gated DeltaNet backbone
    (appendix on linear attention): dv_delta_rule_write for every linear-attention layer."""
    import torch

    import paper_2609_34972_amd as dvl
    from paper_2609_34972_amd import configs

    steps = steps if steps is not None else args.steps
    warmup = warmup if warmup is not None else args.warmup
    dev = torch.device("cuda:0")
    dt = torch.bfloat16 if w.dtype == "bf16" else torch.float32
    log(f"[bench] generating {w.name} inputs for {w.layers} layers on the GPU")
    gen = torch.Generator(device=dev)
    gen.manual_seed(0)
    rn = lambda *s: torch.randn(*s, generator=gen, device=dev, dtype=torch.float32)
    layers = []
    for _ in range(w.layers):
        k = rn(w.B, w.Hk, w.N, w.dk)
        k = (k / k.norm(dim=-1, keepdim=True)).to(dt)
        layers.append({"k": k, "v": rn(w.B, w.Hv, w.N, w.dv).to(dt),
                       "alpha": torch.exp(-0.1 * torch.nn.functional.softplus(rn(w.B, w.Hv, w.N))),
                       "beta": torch.sigmoid(rn(w.B, w.Hv, w.N)),
                       "S": 0.1 * rn(w.B, w.Hv, w.dk, w.dv)})
    ws = torch.empty(dvl.delta_rule_workspace(w.B, w.Hv, w.N, w.dk, w.dv, dt), dtype=torch.uint8,
                     device=dev)

    def step(ev=None):
        for l, x in enumerate(layers):
            if ev is not None:
                dvl.time_kernel(dvl.KERNEL_DELTA_PREP, *ev[l][0])
                dvl.time_kernel(dvl.KERNEL_DELTA_SCAN, *ev[l][1])
            dvl.delta_rule_write(x["k"], x["v"], x["alpha"], x["beta"], x["S"], ws=ws)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    # Steps timed without per-kernel events; the kernels are timed in extra steps afterwards.
    mk = lambda: torch.cuda.Event(enable_timing=True)
    marks = [mk() for _ in range(steps + 1)]
    for s_ in range(steps):
        marks[s_].record()
        step()
    marks[-1].record()
    torch.cuda.synchronize()
    step_ms = [marks[i].elapsed_time(marks[i + 1]) for i in range(steps)]
    hev = HipEvents()
    n_ev = min(steps, 3)
    evs = [[(hev.pair(), hev.pair()) for _ in range(w.layers)] for _ in range(n_ev)]
    for s_ in range(n_ev):
        step(evs[s_])
    torch.cuda.synchronize()
    dvl.time_kernel(dvl.KERNEL_DELTA_PREP)
    dvl.time_kernel(dvl.KERNEL_DELTA_SCAN)
    prep = sum(hev.ms(e[0]) for st in evs for e in st) / (n_ev * w.layers)
    scan = sum(hev.ms(e[1]) for st in evs for e in st) / (n_ev * w.layers)
    hev.close()
    ms = percentiles(step_ms)
    per_layer = ms["median"] / w.layers
    nbytes = configs.bytes_delta_write(w)
    res = {"workload": w.name, "layers": w.layers, "batch": w.B, "tokens": w.N,
           "key_heads": w.Hk, "value_heads": w.Hv, "dk": w.dk, "dv": w.dv,
           "ms_per_step": ms, "ms_per_layer": per_layer, "prep_kernel_ms": prep,
           "scan_kernel_ms": scan,
           "visual_tokens_per_s": w.B * w.N / (ms["median"] * 1e-3),
           "algorithmic_bytes_per_layer": nbytes,
           "gbs": nbytes / (per_layer * 1e-3) / 1e9,
           "hbm_frac": nbytes / (per_layer * 1e-3) / 1e9 / PEAK_HBM_GBS,
           "recurrence_tflops": configs.flops_delta_write(w) / (per_layer * 1e-3) / 1e12}
    del layers, ws
    torch.cuda.empty_cache()
    return res


def run_decode(args, w, layers_timed=None):
    """Decode: one new text token per sequence reading every layer's cached visual and text K/V."""
    import torch

    import paper_2609_34972_amd as dvl
    from paper_2609_34972_amd import configs

    dev = torch.device("cuda:0")
    L = w.L if layers_timed is None else layers_timed
    log(f"[bench] generating decode caches for {L} layers on the GPU")
    gen = torch.Generator(device=dev)
    gen.manual_seed(0)
    rn = lambda *s: torch.randn(*s, generator=gen, device=dev, dtype=torch.float32).to(torch.bfloat16)
    caches = []
    for _ in range(L):
        caches.append({"Q": rn(w.B, 1, w.Hq, w.hd), "Kv": rn(w.B, w.Hkv, w.Nv, w.hd),
                       "Vv": rn(w.B, w.Hkv, w.Nv, w.hd), "Kt": rn(w.B, w.Hkv, w.Nkt, w.hd),
                       "Vt": rn(w.B, w.Hkv, w.Nkt, w.hd)})
    O = torch.empty(w.B, 1, w.Hq, w.hd, dtype=torch.bfloat16, device=dev)
    na = dvl.text_visual_attention_workspace(w.B, w.Hq, w.Hkv, w.hd, w.Nv, 1, w.Nkt)
    ws = torch.empty(max(na, 16), dtype=torch.uint8, device=dev)

    def step(ev=None):
        for l in range(L):
            c = caches[l]
            if ev is not None:
                dvl.time_kernel(dvl.KERNEL_ATTENTION, *ev[l])
            dvl.text_visual_attention(c["Q"], c["Kv"], c["Vv"], c["Kt"], c["Vt"], O, q_pos0=w.q_pos0,
                                      ws=ws)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    # Steps timed without per-kernel events; the kernels are timed in extra steps afterwards.
    mk = lambda: torch.cuda.Event(enable_timing=True)
    t0, t1 = mk(), mk()
    t0.record()
    for s in range(args.steps):
        step()
    t1.record()
    torch.cuda.synchronize()
    ms_step = t0.elapsed_time(t1) / args.steps
    hev = HipEvents()
    n_ev = min(args.steps, 3)
    evs = [[hev.pair() for _ in range(L)] for _ in range(n_ev)]
    for s in range(n_ev):
        step(evs[s])
    torch.cuda.synchronize()
    dvl.time_kernel(dvl.KERNEL_ATTENTION)
    ms_launch = sum(hev.ms(p) for e in evs for p in e) / (n_ev * L)
    hev.close()
    bytes_layer = configs.bytes_attention(w, layers=1)
    gbs = bytes_layer / (ms_launch * 1e-3) / 1e9
    res = {"ms_per_step": ms_step, "layers": L, "ms_per_layer": ms_step / L,
           "kernel_ms_per_layer": ms_launch, "algorithmic_bytes_per_layer": bytes_layer,
           "kernel_gbs": gbs, "kernel_hbm_frac": gbs / PEAK_HBM_GBS,
           "step_gbs": bytes_layer * L / (ms_step * 1e-3) / 1e9,
           "tokens_per_s": w.B / (ms_step * 1e-3)}
    # HBM bytes the kernel really moves (FETCH_SIZE + WRITE_SIZE of a committed counter run)
    # over this run's kernel time, while the counters still match the sources
    tb = stored_traffic(DECODE_TRAFFIC_FILE, ATTN_SOURCES) if w.name == "decode" else None
    res["traffic_bytes_per_layer"] = tb
    res["counter_gbs"] = tb / (ms_launch * 1e-3) / 1e9 if tb else None
    del caches, O, ws
    torch.cuda.empty_cache()
    return res


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only: --gpus {args.gpus} is not supported (the kernels "
              "run on a single MI355X; multi-GPU sharding is a design note, not an implemented path)",
              file=sys.stderr)
        sys.exit(2)
    import torch

    from paper_2609_34972_amd import configs

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    if args.workload in ("gdn_video", "gdn_image"):
        w = configs.GDN_VIDEO if args.workload == "gdn_video" else configs.GDN_IMAGE
        d = run_delta(args, w)
        out = {
            "metric": METRIC, "value": d["visual_tokens_per_s"],
            "unit": f"visual tokens/s written into {w.layers} linear-attention layers",
            "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
            "ms_per_step": d["ms_per_step"]["median"], "higher_is_better": True,
            "scaling": "weak", "vs_baseline": None, "dtype": w.dtype, "data": "synthetic",
            "config": {"workload": w.name, "batch": w.B, "visual_tokens": w.N,
                       "key_heads": w.Hk, "value_heads": w.Hv, "dk": w.dk, "dv": w.dv,
                       "layers": w.layers},
            "roofline": {"bound": "hbm", "kernel": "k_gdr_prep + k_gdr_chain (+ k_gdr_merge)",
                         "achieved": d["gbs"], "peak": PEAK_HBM_GBS, "unit": "GB/s",
                         "frac": d["hbm_frac"], "traffic": None,
                         "algorithmic_bytes_per_launch": d["algorithmic_bytes_per_layer"],
                         "ms_per_launch": d["ms_per_layer"]},
            "delta_write": d,
        }
        out["provenance"] = provenance()
        print(json.dumps(out), flush=True)
        return
    w = configs.get(args.workload)
    if w.decode:
        d = run_decode(args, w)
        out = {
            "metric": METRIC, "value": d["tokens_per_s"], "unit": "decoded tokens/s (32 layers)",
            "n_gpus": 1, "steps": args.steps, "warmup": args.warmup, "ms_per_step": d["ms_per_step"],
            "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
            "data": "synthetic",
            "config": {"workload": w.name, "batch": w.B, "visual_tokens": w.Nv,
                       "text_keys": w.Nkt, "layers": w.L, "q_heads": w.Hq, "kv_heads": w.Hkv,
                       "head_dim": w.hd},
            "roofline": {"bound": "hbm", "kernel": "k_attn_decode", "achieved": d["kernel_gbs"],
                         "peak": PEAK_HBM_GBS, "unit": "GB/s", "frac": d["kernel_hbm_frac"],
                         "traffic": d["traffic_bytes_per_layer"],
                         "algorithmic_bytes_per_launch": d["algorithmic_bytes_per_layer"],
                         "ms_per_launch": d["kernel_ms_per_layer"]},
            "decode": d,
        }
    else:
        out = run_prefill(args, w)
        if w.name == "llava7b" and not args.no_workloads:
            out["workloads"] = {o.name: run_workload_block(args, o)
                                for o in (configs.LLAVA_NEXT, configs.QWEN25VL_VIDEO)}
        if not args.no_decode:
            out["decode"] = run_decode(args, configs.DECODE)
        if not args.no_delta:
            out["delta_write"] = run_delta(args, configs.GDN_VIDEO, steps=5, warmup=1)
    if args.calibrate_copy:
        n = 1 << 30
        src = torch.empty(n, dtype=torch.uint8, device="cuda:0").fill_(1)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        out["calibration_copy_bytes"] = n
        del src, dst
    out["provenance"] = provenance()
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
