"""Benchmark: one device's patch-parallel DiT-XL/2 1024px denoising step.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--share 0.40]

A step is one orch_patch_denoise_step call: the DiT-XL/2 denoiser (28 blocks,
hidden 1152, 16 heads) on a band of token rows of the 64 x 64 token grid
(40% = 26 rows = 1664 queries per branch), attention over all 4096 tokens
(fresh K/V for the band, stale buffer for the rest, refreshed in place),
classifier-free guidance batch 2, and the scheduler update, at the first
post-warm-up step t 780 -> 760 of the 50-step schedule.  Inputs are seeded
and synthetic: random N(0, 0.02) weights, N(0, 1) latent; the stale K/V
buffer is what the synchronous warm-up leaves, every token's K/V of a
full-image step at the previous grid timestep on an independent seeded
latent, computed by the library before timing.

Prints one JSON line: algorithmic TFLOP/s of the step (value), ms per step,
the per-kernel split measured inside the steps (HIP events around every
launch, a second pass after the timed one) with the dominant kernel's
roofline, the HBM-bound kernels at large shapes, the share sweep (10% to
100% bands, and three shares at 2048px; --no-sweep skips it), the CPU oracle
timed on one whole 10% band step, and one compact figure for each adjacent
part (--no-extras skips them): the band's whole tiered sampler schedule
(`schedule`), Algorithm 1 over four virtual devices planned from fixed
speeds (`virtual_devices`) and the U-Net band block on three SDXL-sized
stages (`unet`).  --unet, --schedule and --virtual-devices print only that
figure, timed over --steps passes; --pmc-probe / --pmc-report serve the HBM
counter runs.
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

PEAK_BF16_TFLOPS = 2500.0       # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0
METRIC = "patch-step ms and TFLOP/s vs bf16 MFMA peak, DiT-XL/2 1024px, 1 GPU"
SWEEP_SHARES = (0.10, 0.25, 0.40, 0.65, 1.00)   # elastic band shares of the 1024px grid
SWEEP_SHARES_2048 = (0.125, 0.375, 0.625)         # band shares of the 2048px grid
CPU_SHARE = 0.10                                 # band the oracle is timed on, whole step
PROFILE_ROWS = (4, 8, 16, 32, 64)                # band heights of a device's time profile
MFMA_KERNELS = ("qkv_gemm", "attention", "proj_gemm", "fc1_gemm", "fc2_gemm")

# HBM traffic of the dominant kernel, from two rocprofv3 --pmc runs of
# `bench.py --pmc-probe` (FETCH_SIZE, then WRITE_SIZE) turned into a report by
# `bench.py --pmc-report`; valid only while the kernel's sources are unchanged.
TRAFFIC_REPORT = os.path.join(ROOT, "profiles", "attention_xl1024_band40_traffic.md")
# timed passes of each adjacent part's figure in the default line
EXTRA_PASSES = 3
KERNEL_SOURCES = {
    "attention": ["paper_2509_04719_amd/csrc/k_attention.hip", "paper_2509_04719_amd/csrc/common.h",
                  "paper_2509_04719_amd/csrc/kernels.h", "paper_2509_04719_amd/build.py"],
}
# the attention launch: the main kernel, and the merge of the query tiles it
# cut between workgroups (absent when every tile stays whole)
KERNEL_NAMES = {"attention": ["attn_bf16_mfma_kernel", "attn_merge_kernel"]}
# calibration: the scheduler-update kernel with no unconditional branch and no
# noise reads x and eps and writes out, 4 bytes each per element
CALIB_ELEMS = 64 << 20
CALIB_NAME = "update_vec4_kernel"


def kernel_source_hash(kernel: str) -> str:
    import hashlib
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES[kernel]:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def recorded_traffic(kernel: str):
    """Bytes per launch from the committed counter report, or None when the
    report is missing or the kernel's sources changed since it was taken."""
    try:
        with open(TRAFFIC_REPORT) as f:
            kv = dict(l.strip()[2:].split(": ", 1) for l in f if l.startswith("- ") and ": " in l)
    except OSError:
        return None
    if kv.get("kernel") != kernel or kv.get("source_sha256") != kernel_source_hash(kernel):
        return None
    return float(kv["hbm_bytes_per_launch"])


def pmc_probe(a) -> int:
    """Workload of the counter runs: the calibration stream, then the bench
    step (warm-up and three timed-shape steps)."""
    import numpy as np
    import torch

    from paper_2509_04719_amd import _lib as L
    from paper_2509_04719_amd import schedule as psched
    from seeded_inputs import configs, generate

    dev = "cuda:0"
    xs = torch.randn(CALIB_ELEMS, device=dev)
    es = torch.randn(CALIB_ELEMS, device=dev)
    os_ = torch.empty(CALIB_ELEMS, device=dev)
    for _ in range(3):
        L.scheduler_update(xs, es, None, 1.0, None, 0.9, 0.1, 0.0, os_)
    torch.cuda.synchronize()
    del xs, es, os_
    cfg = configs.get(a.config)
    rows = psched.band_rows(a.share, cfg.R)
    t, tp = configs.headline_timestep_pair(cfg)
    ctx = L.DiTStep(cfg, generate.make_weight_blob(cfg, 0))
    x = torch.from_numpy(generate.make_latent(cfg, 0)).to(dev)
    labels = generate.make_labels(cfg, 0)
    kv = torch.zeros(ctx.stale_kv_bytes() // 2, dtype=torch.bfloat16, device=dev)
    xs = torch.from_numpy(generate.make_stale_latent(cfg, 0)).to(dev)
    full_out = torch.empty((cfg.in_ch, cfg.latent, cfg.latent), device=dev)
    ctx.step(xs, 0, cfg.R, t + cfg.T // cfg.steps, t, labels, cfg.cfg_scale, kv, 1, full_out)
    out = torch.empty((cfg.in_ch, rows * cfg.patch, cfg.latent), device=dev)
    for _ in range(5):
        ctx.step(x, 0, rows, t, tp, labels, cfg.cfg_scale, kv, 1, out)
    torch.cuda.synchronize()
    ctx.close()
    print("pmc probe done", flush=True)
    return 0


def pmc_report(fetch_dir: str, write_dir: str, kernel: str = "attention") -> int:
    """Summarise the two counter runs (FETCH_SIZE, WRITE_SIZE; KiB per
    dispatch) as the traffic report bench.py reads."""
    import csv
    import glob

    def per_dispatch(d, counter):
        # {kernel key: {dispatch: (grid size, counter sum)}}; the calibration
        # dispatches are the update launches with the largest grid (the steps
        # launch the same kernel on the band)
        vals = {}
        for f in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
            for r in csv.DictReader(open(f)):
                if r["Counter_Name"] != counter:
                    continue
                for key in [CALIB_NAME] + KERNEL_NAMES[kernel]:
                    if key in r["Kernel_Name"]:
                        g, v = vals.setdefault(key, {}).get(r["Dispatch_Id"], (int(r["Grid_Size"]), 0.0))
                        vals[key][r["Dispatch_Id"]] = (g, v + float(r["Counter_Value"]))
        out = {}
        for key, disp in vals.items():
            gmax = max(g for g, _ in disp.values())
            keep = [v for g, v in disp.values() if key != CALIB_NAME or g == gmax]
            out[key] = sorted(keep)
        return out

    fetch = per_dispatch(fetch_dir, "FETCH_SIZE")
    write = per_dispatch(write_dir, "WRITE_SIZE")
    med = lambda v: v[len(v) // 2]
    calib_read_kib, calib_write_kib = 8 * CALIB_ELEMS / 1024, 4 * CALIB_ELEMS / 1024
    fscale = calib_read_kib / med(fetch[CALIB_NAME])
    wscale = calib_write_kib / med(write[CALIB_NAME])
    names = [k for k in KERNEL_NAMES[kernel] if k in fetch and k in write]
    fb = sum(med(fetch[k]) for k in names) * fscale * 1024
    wb = sum(med(write[k]) for k in names) * wscale * 1024
    print(f"# HBM traffic of the {kernel} kernel, DiT-XL/2 1024px band step (26 of 64 rows)\n")
    print("Commands (repository root, on the GPU host):\n")
    print("    rocprofv3 --pmc FETCH_SIZE -d <fetch_dir> -o pmc --output-format csv -- python3 bench.py --pmc-probe")
    print("    rocprofv3 --pmc WRITE_SIZE -d <write_dir> -o pmc --output-format csv -- python3 bench.py --pmc-probe")
    print("    python3 bench.py --pmc-report <fetch_dir> <write_dir>\n")
    print(f"Calibration: `{CALIB_NAME}` over {CALIB_ELEMS} fp32 elements reads {8 * CALIB_ELEMS} B and writes "
          f"{4 * CALIB_ELEMS} B; the counters read {med(fetch[CALIB_NAME]):.1f} KiB and "
          f"{med(write[CALIB_NAME]):.1f} KiB per dispatch, so FETCH_SIZE is scaled by {fscale:.4f} and "
          f"WRITE_SIZE by {wscale:.4f}.\n")
    for k in names:
        print(f"Per `{k}` dispatch (median of {len(fetch[k])} / {len(write[k])}): FETCH_SIZE "
              f"{med(fetch[k]):.1f} KiB, WRITE_SIZE {med(write[k]):.1f} KiB.\n")
    print(f"A launch of the {kernel} is one dispatch of each kernel listed (the merge kernel runs only "
          f"where query tiles are cut between workgroups); its bytes are their sum.\n")
    print(f"- kernel: {kernel}")
    print(f"- source_sha256: {kernel_source_hash(kernel)}")
    print(f"- fetch_bytes_per_launch: {fb:.0f}")
    print(f"- write_bytes_per_launch: {wb:.0f}")
    print(f"- hbm_bytes_per_launch: {fb + wb:.0f}")
    return 0


def step_flops(cfg, n_q: int) -> float:
    """Algorithmic FLOPs of one band step (band tokens only; nothing for stale rows)."""
    H, L, B, N = cfg.hidden, cfg.n_blocks, cfg.cfg_batch, cfg.n_kv
    per_branch = n_q * (L * (24 * H * H + 4 * N * H) + 64 * H) + 12 * H * H * L + 4 * H * H
    return float(B * per_branch + 512 * H + 2 * H * H)


def _time_loop(torch, fn, iters: int, warm: int = 3) -> float:
    """Average ms of fn() over `iters` launches, HIP events on the current stream."""
    for _ in range(warm):
        fn()
    torch.cuda.synchronize()
    s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    s.record()
    for _ in range(iters):
        fn()
    e.record()
    torch.cuda.synchronize()
    return s.elapsed_time(e) / iters


def kernel_split(torch, L, cfg, n_q: int, iters: int):
    """Per-kernel average launch time of the step's hot kernels at the
    step's shapes, through the kernel-level entry points."""
    dev = "cuda:0"
    H, F, B, N, heads, d = cfg.hidden, cfg.mlp_hidden, cfg.cfg_batch, cfg.n_kv, cfg.heads, cfg.head_dim
    M = B * n_q
    bf = torch.bfloat16
    g = torch.Generator(device=dev).manual_seed(0)

    def rnd(*shape, dtype=bf, scale=1.0):
        return (torch.randn(*shape, generator=g, device=dev) * scale).to(dtype)

    u = rnd(M, H)
    w_qkv, w_proj, w_fc1, w_fc2 = rnd(3 * H, H, scale=0.02), rnd(H, H, scale=0.02), \
        rnd(F, H, scale=0.02), rnd(H, F, scale=0.02)
    b3, b1, b4 = rnd(3 * H, dtype=torch.float32), rnd(H, dtype=torch.float32), rnd(F, dtype=torch.float32)
    gate = rnd(B, H, dtype=torch.float32, scale=0.03)
    h = rnd(M, H, dtype=torch.float32)
    mlp = rnd(M, F)
    q = rnd(B, heads, n_q, d)
    kv = rnd(B * 2 * N * H, scale=0.7)
    att = torch.empty(M, H, dtype=bf, device=dev)
    mod = rnd(B, 3 * H, dtype=torch.float32, scale=0.1)
    fl = {}
    fl["qkv_gemm"] = (2.0 * M * H * 3 * H, lambda: L.qkv_projection(
        u, B, n_q, H, w_qkv, b3, H, heads, q, kv, 2 * N * H, N, 0, 1))
    wsb = L.attention_workspace_bytes(B, heads, n_q, N, d, 1)
    aws = torch.empty(max(wsb, 1), dtype=torch.uint8, device=dev)
    fl["attention"] = (4.0 * B * n_q * N * H, lambda: L.attention(
        q, kv, 2 * N * H, None, 0, 0, 0, B, heads, n_q, N, d, att, 1, workspace=aws))
    fl["proj_gemm"] = (2.0 * M * H * H, lambda: L.linear(att, M, H, w_proj, H, b1, 2, gate, H, n_q, h, 1))
    fl["fc1_gemm"] = (2.0 * M * H * F, lambda: L.linear(u, M, H, w_fc1, F, b4, 1, None, 0, 1, mlp, 1))
    fl["fc2_gemm"] = (2.0 * M * F * H, lambda: L.linear(mlp, M, F, w_fc2, H, b1, 2, gate, H, n_q, h, 1))
    ln_bytes = 6.0 * M * H
    fl["adaln_layernorm"] = (0.0, lambda: L.layernorm_modulate(h, M, H, n_q, mod, mod[:, H:], 3 * H, u, 1))
    out = {}
    for name, (flops, fn) in fl.items():
        ms = _time_loop(torch, fn, iters)
        rec = {"ms": round(ms, 5)}
        if flops:
            rec["tflops"] = round(flops / ms / 1e9, 1)
            rec["flop_per_launch"] = flops
        else:
            rec["gbs"] = round(ln_bytes / ms / 1e6, 1)
            rec["bytes_per_launch"] = ln_bytes
        out[name] = rec
    return out


def hbm_kernels(torch, L):
    """The HBM-bound elementwise kernels at large synthetic shapes, where
    launch overhead no longer hides the streaming rate: the guided scheduler
    update over 256 Mi elements (x, both branches' eps in, out: 16 B per
    element) and the adaLN LayerNorm over 65536 rows of 1152 (fp32 in, bf16
    out: 6 B per element).  GB/s = algorithmic bytes / average launch time."""
    dev = "cuda:0"
    res = {}
    n = 256 << 20
    x = torch.randn(n, device=dev)
    ec, eu = torch.randn(n, device=dev), torch.randn(n, device=dev)
    out = torch.empty(n, device=dev)
    ms = _time_loop(torch, lambda: L.scheduler_update(x, ec, eu, 1.5, None, 1.2, 0.2, 0.0, out), 10)
    res["scheduler_update_256Mi"] = {"us": round(ms * 1e3, 1), "gbs": round(16 * n / ms / 1e6, 1)}
    del x, ec, eu, out
    rows, H = 65536, 1152
    h = torch.randn(rows, H, device=dev)
    mod = torch.randn(2, 2 * H, device=dev) * 0.1
    u = torch.empty(rows, H, dtype=torch.bfloat16, device=dev)
    ms = _time_loop(torch, lambda: L.layernorm_modulate(h, rows, H, rows // 2, mod[:, :H], mod[:, H:],
                                                       2 * H, u, 1), 10)
    res["layernorm_65536x1152"] = {"us": round(ms * 1e3, 1), "gbs": round(6 * rows * H / ms / 1e6, 1)}
    return res


def step_kernel_split(ctx, cfg, n_q: int, run_step, steps: int):
    """Per-kernel-class average launch time inside the step itself: every
    launch of `steps` steps bracketed by HIP events on the step's stream
    (orch_set_kernel_timing), with the algorithmic work of one launch."""
    H, F, B, N, L = cfg.hidden, cfg.mlp_hidden, cfg.cfg_batch, cfg.n_kv, cfg.n_blocks
    M = B * n_q
    flops = {"qkv_gemm": 2.0 * M * H * 3 * H, "attention": 4.0 * B * n_q * N * H,
             "proj_gemm": 2.0 * M * H * H, "fc1_gemm": 2.0 * M * H * F, "fc2_gemm": 2.0 * M * F * H}
    nbytes = {"layernorm": 6.0 * M * H,                       # fp32 in, bf16 out
              "conditioning": 2.0 * (6 * H * H * L + 2 * H * H),  # adaLN weights streamed
              "update": 16.0 * cfg.in_ch * (n_q // cfg.R) * cfg.patch * cfg.latent}
    ctx.set_kernel_timing(True)
    ctx.kernel_times()
    for _ in range(steps):
        run_step()
    times = ctx.kernel_times()
    ctx.set_kernel_timing(False)
    out = {}
    for k, (ms, n) in times.items():
        if n == 0:
            continue
        avg = ms / n
        rec = {"ms": round(avg, 5), "launches_per_step": n // steps,
               "ms_per_step": round(ms / steps, 4)}
        if k in flops:
            rec["tflops"] = round(flops[k] / avg / 1e9, 1)
            rec["flop_per_launch"] = flops[k]
        if k in nbytes:
            rec["gbs"] = round(nbytes[k] / avg / 1e6, 1)
            rec["bytes_per_launch"] = nbytes[k]
        out[k] = rec
    return out


def sweep_2048(torch, L, steps: int) -> dict:
    """DiT-XL/2 at 2048px (128 token rows, 16384 keys): one band step at each
    of the 1/8, 3/8 and 5/8 shares at the first stride-2 step of the tiered
    schedule, the stale buffer filled by a full-image step first (as the
    1024px bench)."""
    from paper_2509_04719_amd import schedule as psched
    from seeded_inputs import configs, generate

    dev = "cuda:0"
    cfg = configs.get("dit_xl2_2048")
    t, tp = configs.headline_timestep_pair(cfg)
    ctx = L.DiTStep(cfg, generate.make_weight_blob(cfg, 0))
    x = torch.from_numpy(generate.make_latent(cfg, 0)).to(dev)
    labels = generate.make_labels(cfg, 0)
    kv = torch.zeros(ctx.stale_kv_bytes() // 2, dtype=torch.bfloat16, device=dev)
    xs = torch.from_numpy(generate.make_stale_latent(cfg, 0)).to(dev)
    full_out = torch.empty((cfg.in_ch, cfg.latent, cfg.latent), device=dev)
    ctx.step(xs, 0, cfg.R, t + cfg.T // cfg.steps, t, labels, cfg.cfg_scale, kv, 1, full_out)
    del xs, full_out
    res = {}
    for share in SWEEP_SHARES_2048:
        r = psched.band_rows(share, cfg.R)
        o = torch.empty((cfg.in_ch, r * cfg.patch, cfg.latent), device=dev)

        def band_step():
            ctx.step(x, 0, r, t, tp, labels, cfg.cfg_scale, kv, 1, o)
        m = _time_loop(torch, band_step, steps, 2)
        ks = step_kernel_split(ctx, cfg, cfg.n_q(r), band_step, 2)
        res[f"{r}/{cfg.R}"] = {"rows": r, "n_q": cfg.n_q(r), "ms": round(m, 3),
                               "tflops": round(step_flops(cfg, cfg.n_q(r)) / m / 1e9, 1),
                               "attention_tflops": ks["attention"]["tflops"],
                               "attention_frac": round(ks["attention"]["tflops"] / PEAK_BF16_TFLOPS, 4)}
    ctx.close()
    return {"workload": f"{cfg.name}: {cfg.R} token rows, {cfg.n_kv} keys, t {t}->{tp}", "shares": res}


def host_info() -> dict:
    """CPU model, numpy and its BLAS, and the cores this process may use."""
    import platform

    import numpy as np
    model = platform.processor() or "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    blas, threads = "unknown", None
    try:
        from threadpoolctl import threadpool_info
        infos = [i for i in threadpool_info() if i.get("user_api") == "blas"]
        if infos:
            blas = f"{infos[0].get('internal_api')} {infos[0].get('version')}"
            threads = infos[0].get("num_threads")
    except Exception:
        pass
    return {"cpu_model": model, "numpy": np.__version__, "blas": blas, "blas_threads": threads,
            "affinity_cores": len(os.sched_getaffinity(0))}


def cpu_baseline(cfg, blob, x, labels, stale, rb, re, t, tp):
    """The oracle (float64 numpy) timed on one whole band step: every block,
    both guidance branches, the update; no extrapolation."""
    import numpy as np

    from oracle import blob as oblob
    from oracle import dit
    hdr, params = oblob.read_blob(blob, np.float64)
    t0 = time.perf_counter()
    dit.patch_step(hdr, params, x, rb, re, t, tp, labels, cfg.cfg_scale, stale)
    dt = time.perf_counter() - t0
    fl = step_flops(cfg, (re - rb) * cfg.R)
    info = host_info()
    cores = info["blas_threads"] or info["affinity_cores"]
    return {"value": round(fl / dt / 1e12, 5), "unit": "TFLOP/s", "cores": cores, "kind": "oracle",
            "sample": f"{cfg.name} band rows [{rb},{re}) ({re - rb}/{cfg.R}), all {cfg.n_blocks} "
                      f"blocks, both guidance branches and the update, float64 numpy: one whole "
                      f"step of {fl / 1e12:.3f} TFLOP in {dt:.1f} s",
            "ms_per_step": round(dt * 1e3, 1), **info}


def schedule_result(n_passes, cfg, ctx, x, labels, kv, rows, n_q) -> dict:
    """Every executed step of the band's sampler (tiered for configs that use
    it: Algorithm 1's reduced tier, Eq. (2)); x of the band is carried from
    step to step (in place) and the buffer refreshed on executed steps."""
    import torch

    from paper_2509_04719_amd import schedule as psched
    steps = (psched.tiered_schedule(cfg.T, cfg.steps, cfg.warmup) if cfg.tiered
             else psched.plain_schedule(cfg.T, cfg.steps))
    p = cfg.patch
    out = torch.empty((cfg.in_ch, rows * p, cfg.latent), device=x.device)
    total_flops = step_flops(cfg, n_q) * len(steps)

    def sampler():
        for st in steps:
            ctx.step(x, 0, rows, st.t, st.t_prev, labels, cfg.cfg_scale, kv, int(st.refresh), out)
            x[:, 0:rows * p].copy_(out)

    sampler()                                          # warm-up pass
    torch.cuda.synchronize()
    s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    s.record()
    for _ in range(n_passes):
        sampler()
    e.record()
    torch.cuda.synchronize()
    ms = s.elapsed_time(e) / n_passes
    return {"metric": "full-schedule ms of one device's band sampler", "value": round(ms, 3),
           "unit": "ms", "n_gpus": 1, "steps": n_passes, "warmup": 1,
           "ms_per_step": round(ms / len(steps), 4), "higher_is_better": False,
           "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
           "config": {"workload": f"{cfg.name}: band {rows}/{cfg.R} rows, {len(steps)} executed "
                                  f"steps ({'tiered: warm-up ' + str(cfg.warmup) + ', then stride 2' if cfg.tiered else 'plain'})",
                      "executed_steps": len(steps), "n_q": n_q, "kv_len": cfg.n_kv},
           "tflops": round(total_flops / ms / 1e9, 1)}


def run_schedule(a, cfg, ctx, x, labels, kv, rows, n_q) -> int:
    print(json.dumps(schedule_result(a.steps, cfg, ctx, x, labels, kv, rows, n_q)), flush=True)
    ctx.close()
    return 0


def virtual_devices_result(a, cfg, ctx, x, labels, n_passes) -> dict:
    """Algorithm 1 on virtual devices: the device planner (Eq. (2), Eq. (3))
    turns the device speeds into step counts and token rows, then the
    library's sampler runs every band's whole trajectory on this GPU."""
    import torch

    from paper_2509_04719_amd import _lib as L
    from paper_2509_04719_amd import schedule as psched
    from seeded_inputs import configs

    profile = None
    if a.occupancy:
        # Speeds from inference time profiles (§V-A): this GPU's band-step
        # times over band heights; a virtual device with a co-tenant taking a
        # share rho of it runs each step 1 / (1 - rho) times longer.
        occ = [float(v) for v in a.occupancy.split(",")]
        kv_p = torch.zeros(ctx.stale_kv_bytes() // 2, dtype=torch.bfloat16, device=x.device)
        t, tp = configs.headline_timestep_pair(cfg)
        base = []
        for r in PROFILE_ROWS:
            if r > cfg.R:
                continue
            o = torch.empty((cfg.in_ch, r * cfg.patch, cfg.latent), device=x.device)
            m = _time_loop(torch, lambda: ctx.step(x, 0, r, t, tp, labels, cfg.cfg_scale, kv_p, 1, o),
                           5, 2)
            base.append((r, m))
        del kv_p
        profiles = [[(r, m / (1.0 - o)) for r, m in base] for o in occ]
        ref = max(1, round(cfg.R / len(occ)))
        speeds = L.speeds_from_profiles(profiles, ref)
        profile = {"band_rows_ms": [[r, round(m, 4)] for r, m in base], "occupancy": occ,
                   "ref_rows": ref, "speeds": [round(v, 4) for v in speeds]}
        print(f"# profiled speeds: {json.dumps(profile)}", flush=True)
    else:
        speeds = [float(v) for v in a.speeds.split(",")]
    steps, rows = L.plan_devices(speeds, a.m_base, a.m_warmup, a.thr_a, a.thr_b, cfg.R)
    splits, tiers = [0], []
    for st, r in zip(steps, rows):
        if st and r:
            splits.append(splits[-1] + r)
            tiers.append(0 if st == a.m_base else 1)
    grid = psched.grid_desc(cfg.T, a.m_base)
    # algorithmic work: warm-up steps over every row, then per interval one
    # band step per tier-1 band and two per tier-0 band (one at the end if a
    # single grid step is left)
    flops = a.m_warmup * step_flops(cfg, cfg.n_q(cfg.R))
    m = a.m_warmup
    while m < a.m_base:
        two = m + 2 <= a.m_base
        for i, tier in enumerate(tiers):
            n = 2 if (tier == 0 and two) else 1
            flops += n * step_flops(cfg, cfg.n_q(splits[i + 1] - splits[i]))
        m += 2 if two else 1
    n_kv = ctx.stale_kv_bytes()
    kv_a = torch.empty(n_kv, dtype=torch.uint8, device=x.device)
    kv_b = torch.empty(n_kv, dtype=torch.uint8, device=x.device)
    lat = x.clone()

    def sample():
        lat.copy_(x)
        ctx.sample_patch_parallel(lat, splits, tiers, grid, a.m_warmup, labels, cfg.cfg_scale,
                                  kv_a, kv_b)

    sample()                                           # warm-up pass
    torch.cuda.synchronize()
    s, e = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    s.record()
    for _ in range(n_passes):
        sample()
    e.record()
    torch.cuda.synchronize()
    ms = s.elapsed_time(e) / n_passes
    return {"metric": "ms per image of the patch-parallel sampler on virtual devices", "value": round(ms, 2),
           "unit": "ms", "n_gpus": 1, "steps": n_passes, "warmup": 1, "higher_is_better": False,
           "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
           "config": {"workload": f"{cfg.name}: {len(tiers)} virtual devices, speeds "
                                  f"{[round(v, 4) for v in speeds]}, M_base {a.m_base}, M_warmup "
                                  f"{a.m_warmup}, a {a.thr_a}, b {a.thr_b}",
                      "device_steps": steps, "device_rows": rows, "row_splits": splits,
                      "tiers": tiers, "speed_profile": profile},
           "tflops": round(flops / ms / 1e9, 1)}


def run_virtual_devices(a, cfg, ctx, x, labels) -> int:
    print(json.dumps(virtual_devices_result(a, cfg, ctx, x, labels, a.steps)), flush=True)
    ctx.close()
    return 0


def unet_result(n_iters: int, with_cpu: bool) -> dict:
    """The U-Net band block (GroupNorm -> SiLU -> conv3x3 with stale halo rows
    and stale group statistics) on the three stages of an SDXL-sized U-Net at
    1024px (128 x 128 x 320, 64 x 64 x 640, 32 x 32 x 1280): ms per call and
    the convolution's TFLOP/s per band (an interior 1/8, the 14/32 head, the
    18/32 tail and every row)."""
    import numpy as np
    import torch

    from paper_2509_04719_amd import _lib as L
    from seeded_inputs import configs, generate

    dev = "cuda:0"
    stages = {}
    for cfg in (configs.UNET_SDXL_1024, configs.UNET_SDXL_1024_S2, configs.UNET_SDXL_1024_S3):
        H, W, C, Co, G = cfg.height, cfg.width, cfg.channels, cfg.out_channels, cfg.groups
        shape = L.unet_shape(cfg)
        pr = generate.make_unet_params(cfg, 0)
        x = torch.from_numpy(generate.make_unet_input(cfg, 0)).to(dev)
        gamma, beta, bias = (torch.from_numpy(pr[k]).to(dev) for k in ("gamma", "beta", "bias"))
        wt = torch.from_numpy(pr["weight_bits"].view(np.int16)).to(dev).view(torch.bfloat16)
        act = torch.zeros((H, W, C), dtype=torch.bfloat16, device=dev)
        sums = torch.zeros((H, G, 2), device=dev)
        bands = [(7 * H // 16, 9 * H // 16), (0, 14 * H // 32), (14 * H // 32, H), (0, H)]
        # short bands split the taps over more workgroups (fp32 partials): the
        # workspace is sized for every band height used
        wsb = max(L.unet_conv_workspace_bytes(shape, re - rb) for rb, re in bands)
        ws = torch.empty(wsb, dtype=torch.uint8, device=dev)
        full = torch.empty((H, W, Co), device=dev)
        L.unet_conv_band(shape, 0, H, x, gamma, beta, wt, bias, act, sums, 1, full, ws)   # fill buffers
        res = {}
        for rb, re in bands:
            r = re - rb
            xb = x[rb:re].contiguous()
            o = torch.empty((r, W, Co), device=dev)
            ms = _time_loop(torch, lambda: L.unet_conv_band(shape, rb, re, xb, gamma, beta, wt, bias,
                                                            act, sums, 1, o, ws), n_iters)
            fl = 2.0 * r * W * Co * 9 * C
            res[f"[{rb},{re})"] = {"rows": r, "ms": round(ms, 4), "conv_tflops": round(fl / ms / 1e9, 1)}
        stages[cfg.name] = {"shape": f"{H}x{W}x{C}, {G} groups -> {Co}", "bands": res}
        del x, wt, act, sums, ws, full
    # the dominant kernel is the convolution; its rate here is the convolution's
    # FLOPs over the whole call (GroupNorm launches included), a lower bound
    s1 = stages[configs.UNET_SDXL_1024.name]["bands"]
    full_band = s1[f"[0,{configs.UNET_SDXL_1024.height})"]
    roofline = {"kernel": "conv3x3_mfma (whole call timed)", "bound": "mfma",
                "achieved": full_band["conv_tflops"], "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                "frac": round(full_band["conv_tflops"] / PEAK_BF16_TFLOPS, 4),
                "workload": f"{configs.UNET_SDXL_1024.name}, every row"}
    out = {"metric": "U-Net band block ms (GroupNorm, SiLU, conv3x3), SDXL-sized stages at 1024px",
           "unit": "ms", "stages": stages, "roofline": roofline}
    if with_cpu:
        out["cpu_baseline"] = unet_cpu_baseline(configs.UNET_SDXL_1024, 0, configs.UNET_SDXL_1024.height)
    return out


def run_unet(a) -> int:
    print(json.dumps(unet_result(a.steps, not a.no_cpu_baseline)), flush=True)
    return 0


def unet_cpu_baseline(cfg, rb, re):
    """The oracle (float64 numpy) timed on one U-Net band call: the group
    statistics from fresh and stale sums, GroupNorm, SiLU, the convolution."""
    import numpy as np

    from oracle import unet
    from oracle.blob import bf16_to_float
    from seeded_inputs import generate
    pr = generate.make_unet_params(cfg, 0)
    params = {"gamma": pr["gamma"].astype(np.float64), "beta": pr["beta"].astype(np.float64),
              "weight": bf16_to_float(pr["weight_bits"]).astype(np.float64),
              "bias": pr["bias"].astype(np.float64)}
    x = generate.make_unet_input(cfg, 0).astype(np.float64)
    stale_act = np.zeros((cfg.height, cfg.width, cfg.channels))
    stale_sums = np.ones((cfg.height, cfg.groups, 2))
    times = []
    for _ in range(3):
        t0 = time.perf_counter()
        unet.band_step(params, x[rb:re], cfg.height, rb, re, cfg.groups, stale_act, stale_sums, 1e-5)
        times.append(time.perf_counter() - t0)
    dt = sorted(times)[1]
    fl = 2.0 * (re - rb) * cfg.width * cfg.out_channels * 9 * cfg.channels
    info = host_info()
    cores = info["blas_threads"] or info["affinity_cores"]
    return {"value": round(fl / dt / 1e12, 5), "unit": "TFLOP/s", "cores": cores, "kind": "oracle",
            "sample": f"{cfg.name} band rows [{rb},{re}) ({re - rb}/{cfg.height}), float64 numpy: "
                      f"median of three calls of {fl / 1e9:.2f} GFLOP (convolution), {dt:.2f} s each",
            "ms_per_call": round(dt * 1e3, 1), **info}


def main(argv=None) -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=30)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--config", default="dit_xl2_1024")
    ap.add_argument("--share", type=float, default=0.40)
    ap.add_argument("--kernel-iters", type=int, default=20)
    ap.add_argument("--op-split", action="store_true",
                    help="also time each hot kernel alone through the kernel-level entry points")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-sweep", action="store_true",
                    help="skip the share sweep (its other band shapes would mix into a "
                         "profiler's per-kernel averages)")
    ap.add_argument("--sweep-steps", type=int, default=10)
    ap.add_argument("--schedule", action="store_true",
                    help="time the whole sampler schedule of the band instead of one step "
                         "(the tiered schedule for configs that use it)")
    ap.add_argument("--virtual-devices", action="store_true",
                    help="time the whole patch-parallel sampler over virtual devices planned "
                         "from --speeds (Algorithm 1 on this GPU)")
    ap.add_argument("--speeds", default="1.0,1.0,0.6,0.6")
    ap.add_argument("--occupancy", default="",
                    help="with --virtual-devices: derive the speeds from this GPU's measured "
                         "band-step times, each virtual device slowed by a co-tenant taking "
                         "the given share (comma list)")
    ap.add_argument("--m-base", type=int, default=50)
    ap.add_argument("--m-warmup", type=int, default=10)
    ap.add_argument("--thr-a", type=float, default=0.75)
    ap.add_argument("--thr-b", type=float, default=0.25)
    ap.add_argument("--unet", action="store_true",
                    help="time the U-Net band block (SDXL first stage at 1024px) instead")
    ap.add_argument("--no-extras", action="store_true",
                    help="skip the tiered-schedule, virtual-device and U-Net figures of the default line")
    ap.add_argument("--pmc-probe", action="store_true",
                    help="run the workload of the HBM counter runs and exit")
    ap.add_argument("--pmc-report", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="print the traffic report from two counter runs and exit")
    a = ap.parse_args(argv)
    if a.pmc_report:
        return pmc_report(*a.pmc_report)
    if a.gpus != 1:
        print(f"bench.py runs on one GPU only: this build has no multi-GPU path "
              f"(asked for --gpus {a.gpus}).", file=sys.stderr)
        return 2

    import numpy as np
    import torch

    from paper_2509_04719_amd import _lib as L     # raises if liborch.so is missing
    from paper_2509_04719_amd import schedule as psched
    from seeded_inputs import configs, generate

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 1
    if a.pmc_probe:
        return pmc_probe(a)
    if a.unet:
        return run_unet(a)
    dev = "cuda:0"
    cfg = configs.get(a.config)
    rows = psched.band_rows(a.share, cfg.R)
    rb, re = 0, rows
    n_q = cfg.n_q(rows)
    t, tp = configs.headline_timestep_pair(cfg)
    print(f"# bench {cfg.name}: band [{rb},{re}) of {cfg.R} rows, n_q {n_q}, t {t}->{tp}", flush=True)

    blob = generate.make_weight_blob(cfg, 0)
    ctx = L.DiTStep(cfg, blob)
    x_np = generate.make_latent(cfg, 0)
    labels = generate.make_labels(cfg, 0)
    x = torch.from_numpy(x_np).to(dev)
    p = cfg.patch
    # The stale buffer as Algorithm 1's synchronous warm-up leaves it: every
    # token's K/V of a full-image step at the previous grid timestep, on an
    # independent seeded latent.
    kv = torch.zeros(ctx.stale_kv_bytes() // 2, dtype=torch.bfloat16, device=dev)
    xs = torch.from_numpy(generate.make_stale_latent(cfg, 0)).to(dev)
    full_out = torch.empty((cfg.in_ch, cfg.latent, cfg.latent), device=dev)
    ctx.step(xs, 0, cfg.R, t + cfg.T // cfg.steps, t, labels, cfg.cfg_scale, kv, 1, full_out)
    del xs, full_out
    stale_np = generate.make_stale_kv(cfg, 0)      # oracle timing input (values do not matter)
    out = torch.empty((cfg.in_ch, rows * p, cfg.latent), device=dev)

    def one():
        ctx.step(x, rb, re, t, tp, labels, cfg.cfg_scale, kv, 1, out)

    if a.schedule:
        return run_schedule(a, cfg, ctx, x, labels, kv, rows, n_q)
    if a.virtual_devices:
        return run_virtual_devices(a, cfg, ctx, x, labels)

    for _ in range(a.warmup):
        one()
    torch.cuda.synchronize()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(a.steps + 1)]
    ev[0].record()
    for i in range(a.steps):
        one()
        ev[i + 1].record()
    torch.cuda.synchronize()
    per = [ev[i].elapsed_time(ev[i + 1]) for i in range(a.steps)]
    total_ms = ev[0].elapsed_time(ev[-1])
    ms = total_ms / a.steps
    flops = step_flops(cfg, n_q)
    tflops = flops / ms / 1e9
    print(f"# step {ms:.3f} ms (median {float(np.median(per)):.3f}), {tflops:.1f} TFLOP/s", flush=True)

    split = step_kernel_split(ctx, cfg, n_q, one, a.steps)
    dom = max(split, key=lambda k: split[k]["ms_per_step"])
    d = split[dom]
    mfma_names = [k for k in MFMA_KERNELS if k in split]
    mfma_flops = sum(split[k]["flop_per_launch"] * split[k]["launches_per_step"] for k in mfma_names)
    mfma_ms = sum(split[k]["ms_per_step"] for k in mfma_names)
    traffic = recorded_traffic(dom) if dom in KERNEL_SOURCES else None
    roofline = {"kernel": dom, "bound": "mfma", "achieved": d["tflops"], "peak": PEAK_BF16_TFLOPS,
                "unit": "TFLOP/s", "frac": round(d["tflops"] / PEAK_BF16_TFLOPS, 4),
                "traffic": None if traffic is None else round(traffic),
                "traffic_unit": "bytes per launch (FETCH_SIZE + WRITE_SIZE, calibrated)",
                "flop_per_launch": d["flop_per_launch"], "ms_per_launch": d["ms"],
                "measured": "HIP events around each launch inside the timed steps"}
    print(f"# kernels: {json.dumps(split)}", flush=True)
    if a.op_split:
        print(f"# kernel-level entry points: {json.dumps(kernel_split(torch, L, cfg, n_q, a.kernel_iters))}",
              flush=True)

    hbm = hbm_kernels(torch, L)
    print(f"# HBM-bound kernels at large shapes: {json.dumps(hbm)}", flush=True)

    sweep, sweep2048 = {}, {}
    if not a.no_sweep:
        for share in SWEEP_SHARES:
            r = psched.band_rows(share, cfg.R)
            o = torch.empty((cfg.in_ch, r * p, cfg.latent), device=dev)

            def band_step():
                ctx.step(x, 0, r, t, tp, labels, cfg.cfg_scale, kv, 1, o)
            m = _time_loop(torch, band_step, a.sweep_steps, 2)
            ks = step_kernel_split(ctx, cfg, cfg.n_q(r), band_step, 3)
            ag = [k for k in MFMA_KERNELS if k in ks]
            ag_fl = sum(ks[k]["flop_per_launch"] * ks[k]["launches_per_step"] for k in ag)
            ag_ms = sum(ks[k]["ms_per_step"] for k in ag)
            sweep[f"{share:.0%}"] = {
                "rows": r, "n_q": cfg.n_q(r), "ms": round(m, 3),
                "tflops": round(step_flops(cfg, cfg.n_q(r)) / m / 1e9, 1),
                "frac_of_bf16_peak": round(step_flops(cfg, cfg.n_q(r)) / m / 1e9 / PEAK_BF16_TFLOPS, 4),
                "attn_gemm_tflops": round(ag_fl / ag_ms / 1e9, 1),
                "attn_gemm_frac": round(ag_fl / ag_ms / 1e9 / PEAK_BF16_TFLOPS, 4),
                "attention_tflops": ks["attention"]["tflops"]}
        print(f"# sweep: {json.dumps(sweep)}", flush=True)
        sweep2048 = sweep_2048(torch, L, a.sweep_steps)
        print(f"# sweep 2048px: {json.dumps(sweep2048)}", flush=True)

    # the adjacent parts, one compact figure each (after the sweep: the
    # schedule pass carries the band's latent forward in place)
    extras = {}
    if not a.no_extras:
        extras["schedule"] = schedule_result(EXTRA_PASSES, cfg, ctx, x, labels, kv, rows, n_q)
        print(f"# tiered schedule: {json.dumps(extras['schedule'])}", flush=True)
        extras["virtual_devices"] = virtual_devices_result(a, cfg, ctx, x, labels, EXTRA_PASSES)
        print(f"# virtual devices: {json.dumps(extras['virtual_devices'])}", flush=True)
        extras["unet"] = unet_result(EXTRA_PASSES * 5, False)
        print(f"# U-Net band block: {json.dumps(extras['unet'])}", flush=True)

    cpu = None
    if not a.no_cpu_baseline:
        r10 = psched.band_rows(CPU_SHARE, cfg.R)
        cpu = cpu_baseline(cfg, blob, x_np, labels, stale_np, 0, r10, t, tp)
        print(f"# cpu baseline: {json.dumps(cpu)}", flush=True)

    res = {
        "metric": METRIC, "value": round(tflops, 2), "unit": "TFLOP/s", "n_gpus": 1,
        "steps": a.steps, "warmup": a.warmup, "ms_per_step": round(ms, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": f"{cfg.name}: DiT-XL/2 {cfg.latent * 8}px band step, {rows}/{cfg.R} token rows "
                               f"({a.share:.0%}), {n_q} queries x {cfg.n_kv} keys, CFG batch "
                               f"{cfg.cfg_batch}, t {t}->{tp}, stale K/V refreshed",
                   "global_batch": cfg.cfg_batch, "seq_len": n_q, "kv_len": cfg.n_kv,
                   "parallelism": "none (one device's band)"},
        "frac_of_bf16_peak": round(tflops / PEAK_BF16_TFLOPS, 4),
        "step_ms_median": round(float(np.median(per)), 4),
        "step_ms_p10_p90": [round(float(np.percentile(per, 10)), 4), round(float(np.percentile(per, 90)), 4)],
        "attn_gemm_tflops": round(mfma_flops / mfma_ms / 1e9, 1),
        "attn_gemm_ms_per_step": round(mfma_ms, 4),
        "attn_gemm_frac": round(mfma_flops / mfma_ms / 1e9 / PEAK_BF16_TFLOPS, 4),
        "roofline": roofline,
        "kernels": split,
        "hbm_kernels": hbm,
        "share_sweep": sweep,
        "share_sweep_2048": sweep2048,
        "cpu_baseline": cpu,
        **extras,
    }
    print(json.dumps(res), flush=True)
    ctx.close()
    return 0


if __name__ == "__main__":
    sys.exit(main())
