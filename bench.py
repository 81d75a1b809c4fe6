#!/usr/bin/env python3
"""Throughput of the DAVET hot path on one MI355X.

One bench "step" is one full pass of the hot path over one batch: the
evidence views are built once, then the whole T-step denoising loop runs
(level choice, assembly, layer stack, vocabulary head, commitment) through
``davet_run_schedule``.  ``value`` is denoising steps per second (T times the
loops timed, over the wall time of the timed region), with every input
already resident in HBM.

Defaults: the 32-layer 8B-shaped bf16 stack (d=4096, 32 heads x 128,
SwiGLU 12288, vocab 126464, ~16 GB of weights; four 27x27 crops = 2916
visual tokens, pyramid 2916/784/196; prompt 48, response 128; 64 steps
committing 2 per step; a seeded i.i.d. view level per step).  ``--config``
picks another workload (1 tiny fp32, 2 one layer with one crop, 3 one layer
with five crops, 5 ragged batch of 16).  After the main measurement the
one-layer workloads 2, 3 and 5 are timed briefly as well (``--also``) and
reported under ``other_workloads``.

Also reported, in the same JSON line:
  roofline      the dominant kernel class: algorithmic work per launch
                divided by its mean launch time, timed with HIP events around
                every launch on the library's stream inside the timed region
  cpu_baseline  the CPU oracle timed on this host on a bounded sample (one
                oracle step per view level the schedule uses, extrapolated to
                the schedule)
"""

import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0      # MI355X dense bf16 matrix peak
PEAK_FP32_TFLOPS = 157.3       # fp32 vector peak
PEAK_HBM_GBS = 8000.0


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5,
                    help="timed passes of the full T-step loop")
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--config", type=int, default=4)
    ap.add_argument("--also", default="2,3,5",
                    help="comma-separated workloads timed briefly after the "
                         "main one and reported under other_workloads "
                         "('' for none)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-kernel-timing", action="store_true",
                    help="skip the per-launch HIP events")
    ap.add_argument("--cpu-layers", type=int, default=1,
                    help="layers the CPU oracle runs (extrapolated beyond)")
    ap.add_argument("--mode", choices=["f16", "bf16"], default="f16",
                    help="16-bit operand format for a bf16 model (f16: its "
                         "weights rounded to fp16, exact for 2^-17 <= |w|; "
                         "default.  bf16: bf16 activations into the matrix "
                         "cores, outside the 1e-2 logits tolerance beyond a "
                         "few layers: measured 2.2e-2 at 32)")
    ap.add_argument("--head-layout", choices=["tiled", "rows"],
                    default="tiled",
                    help="vocabulary-head weight layout of a 16-bit model "
                         "(tiled: davet_pack_head at setup; default)")
    ap.add_argument("--mixed-stride", type=int, default=0, metavar="S",
                    help="middle level = the mixed view (coarse tokens plus "
                         "the raw-token lattice of stride S) instead of the "
                         "middle pooling level")
    ap.add_argument("--realizer", choices=["pool", "prune", "merge"],
                    default="pool",
                    help="evidence realizer building the levels (pool: the "
                         "paper's default; prune: nested top-n by L1 norm; "
                         "merge: single-linkage similarity merging)")
    ap.add_argument("--schedule", choices=["config", "policy"],
                    default="config",
                    help="level schedule: the workload's own (config) or the "
                         "allocation policy with the per-sample demand of the "
                         "sample's operation category")
    ap.add_argument("--crossing", action="store_true",
                    help="policy schedules: also time the same levels as a "
                         "fixed schedule and report the per-step cost of the "
                         "policy's device-to-host handshake")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only stream MIB MiB of fp32 through a plain "
                         "elementwise copy (y = x * 1) five times and exit: "
                         "the known-size reference for HBM byte counters")
    ap.add_argument("--views-probe", action="store_true",
                    help="only build the pooled evidence views of one, four "
                         "and five 27x27 crops (d = 4096, fp16, K = 3) 20 "
                         "times each and exit: the launches the view-build "
                         "profile summarises")
    return ap.parse_args()


def views_probe():
    """davet_build_views at the 8B shape: one, four and five 27x27 crops of
    seeded random fp16 encodings, 20 launches per geometry."""
    import torch
    import paper_2608_01821_amd as dv
    gen = torch.Generator(device="cuda").manual_seed(0)
    for crops in (1, 4, 5):
        g = dv.ViewGeom(crops, 27, 4096, 3, dv.DAVET_F16, 0, 0)
        sizes = dv.davet_view_sizes(g)
        v = torch.randn(crops * 729, 4096, device="cuda",
                        generator=gen).half().view(torch.int16)
        levels = [torch.empty((sizes[l], 4096), dtype=torch.int16,
                              device="cuda") for l in range(2)]
        for _ in range(20):
            dv.davet_build_views(g, v, levels)
        torch.cuda.synchronize()
        print(json.dumps({"views_probe_crops": crops, "sizes": sizes,
                          "launches": 20}), flush=True)


def copy_calibration(mib):
    """Five launches of a plain copy of known size: each reads and writes
    exactly ``mib`` MiB, so byte counters read on it give the scale factor
    between counter units and bytes."""
    import torch
    n = (mib << 20) // 4
    x = torch.ones(n, dtype=torch.float32, device="cuda")
    y = torch.empty_like(x)
    for _ in range(5):
        torch.mul(x, 1.0, out=y)
    torch.cuda.synchronize()
    print(json.dumps({"copy_calibration_bytes_read": n * 4,
                      "copy_calibration_bytes_written": n * 4,
                      "launches": 5}), flush=True)


REALIZERS = {"pool": 0, "prune": 1, "merge": 2}


def setup(cfg, mode, head_layout="tiled", mixed_stride=0, realizer="pool"):
    import numpy as np
    import torch

    import paper_2608_01821_amd as dv
    import synth

    t0 = time.time()
    bf = cfg.dtype == "bf16"
    dtype = {"f16": dv.DAVET_F16, "bf16": dv.DAVET_BF16}[mode] if bf \
        else dv.DAVET_F32

    def dev(bits):
        """Upload; a bf16 tensor in fp16 mode is converted on the device."""
        if bits.dtype != np.uint16:
            return torch.from_numpy(bits).cuda()
        t = torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).cuda()
        if dtype == dv.DAVET_F16:
            out = torch.empty_like(t)
            dv.davet_convert(t, dv.DAVET_BF16, out, dv.DAVET_F16)
            torch.cuda.synchronize()
            return out
        return t

    layers = []
    for li in range(cfg.n_layers):
        lw = synth.gen_layer_weights(cfg, li, as_bits=bf)
        layers.append({k: dev(v) for k, v in lw.items()})
        del lw
    embed = dev(synth.gen_embed(cfg, as_bits=bf))
    head = dev(synth.gen_head(cfg, as_bits=bf))
    layout = dv.DAVET_HEAD_ROWS
    if bf and head_layout == "tiled":
        # model-load transform: the vocabulary head in the tiled layout the
        # head kernel streams in order (logits bit-identical to row-major)
        tiled = torch.empty(dv.davet_head_tiled_elems(cfg.vocab, cfg.d),
                            dtype=torch.int16, device="cuda")
        dv.davet_pack_head(head, tiled, cfg.vocab, cfg.d, dtype)
        torch.cuda.synchronize()
        head, layout = tiled, dv.DAVET_HEAD_TILED
    W = dv.Weights(embed, head, layers, head_layout=layout)
    s = synth.gen_sample(cfg, as_bits=bf)
    n = cfg.n_seqs
    geoms, visual, view_bufs, sizes = [], [], [], []
    tdt = torch.int16 if bf else torch.float32
    for i in range(n):
        g = dv.ViewGeom(s["n_crops"][i], cfg.grid, cfg.d, cfg.K, dtype,
                        mixed_stride, REALIZERS[realizer])
        sz = dv.davet_view_sizes(g)
        geoms.append(g)
        sizes.append(sz)
        visual.append(dev(s["visual"][i]))
        for lv in range(cfg.K - 1):
            view_bufs.append(torch.empty((sz[lv], cfg.d), dtype=tdt,
                                         device="cuda"))
    prompt = torch.from_numpy(np.concatenate(s["prompts"])).cuda()
    cu = [0]
    for p in s["prompts"]:
        cu.append(cu[-1] + len(p))
    L = cfg.resp_len
    mcfg = dv.ModelCfg(cfg.n_layers, cfg.d, cfg.n_heads, cfg.head_dim, cfg.ffn,
                       cfg.vocab, cfg.mask_id, cfg.rms_eps, cfg.rope_theta,
                       dtype)
    max_tokens = sum(sz[-1] for sz in sizes) + cu[-1] + n * L
    ws = torch.empty(dv.davet_workspace_bytes(mcfg, max_tokens, n, L),
                     dtype=torch.uint8, device="cuda")
    ids = torch.full((n * L,), cfg.mask_id, dtype=torch.int32, device="cuda")
    msk = torch.ones((n * L,), dtype=torch.uint8, device="cuda")
    pols, fixed = None, None
    if cfg.schedule == "policy":
        p = cfg.policy
        pols = [dv.Policy(p["B"], p["rho"], p["alpha"],
                          dv.davet_demand_prior(c), 1 if p["early"] else 0,
                          cfg.K) for c in s["categories"]]
    else:
        fixed = s["schedule"]
    torch.cuda.synchronize()
    log("setup %.1f s (weights + inputs on device, workspace %.2f GB)"
        % (time.time() - t0, ws.numel() / 1e9))
    return dict(dv=dv, W=W, mcfg=mcfg, geoms=geoms, visual=visual,
                view_bufs=view_bufs, prompt=prompt, cu=cu, L=L, ids=ids,
                msk=msk, ws=ws, pols=pols, fixed=fixed, sizes=sizes,
                sample=s, mixed_stride=mixed_stride, realizer=realizer)


def run_loop(cfg, st):
    st["ids"].fill_(cfg.mask_id)
    st["msk"].fill_(1)
    return st["dv"].davet_run_schedule(
        st["mcfg"], st["W"], st["geoms"], st["visual"], st["view_bufs"],
        st["prompt"], st["cu"], st["L"], cfg.steps, cfg.k, st["pols"],
        st["fixed"], st["ids"], st["msk"], st["ws"])


def work_per_loop(cfg, st, levels):
    """Algorithmic work of one loop per kernel class: flops for matrix work,
    bytes for the streaming kernels (views, head weight stream)."""
    n, T, L, d, F, V = (cfg.n_seqs, cfg.steps, cfg.resp_len, cfg.d, cfg.ffn,
                        cfg.vocab)
    es = 2 if cfg.dtype == "bf16" else 4
    w = {k: 0.0 for k in ("gemm_qkv", "gemm_o", "gemm_gateup", "gemm_down",
                          "attention", "head_gemm_flops", "head_gemm_bytes",
                          "views_bytes", "realizer_keys_bytes")}
    for t in range(T):
        ntot = 0
        rows = 0
        for s in range(n):
            lv = levels[s * T + t]
            N = st["sizes"][s][lv] + (st["cu"][s + 1] - st["cu"][s]) + L
            ntot += N
            w["attention"] += cfg.n_layers * 4.0 * N * N * d
            rows += max(0, L - t * cfg.k)
        w["gemm_qkv"] += cfg.n_layers * 2.0 * ntot * d * 3 * d
        w["gemm_o"] += cfg.n_layers * 2.0 * ntot * d * d
        w["gemm_gateup"] += cfg.n_layers * 2.0 * ntot * d * 2 * F
        w["gemm_down"] += cfg.n_layers * 2.0 * ntot * F * d
        w["head_gemm_flops"] += 2.0 * rows * d * V
        w["head_gemm_bytes"] += float(V * d * es + rows * d * es)
    rz = st.get("realizer", "pool")
    for s in range(n):
        sz = st["sizes"][s]
        c, G = st["sample"]["n_crops"][s], cfg.grid
        if rz == "pool":
            # v read once, every pooled level written once
            w["views_bytes"] += float((sz[-1] + sum(sz[:-1])) * d * es)
            continue
        # keys: v read once, one float64 per token (prune) or edge (merge)
        n_keys = sz[-1] if rz == "prune" else c * 2 * G * (G - 1)
        w["realizer_keys_bytes"] += float(sz[-1] * d * es + 8 * n_keys)
        # level rows: every member row read, every level token written
        members = sum(sz[:-1]) if rz == "prune" else (cfg.K - 1) * sz[-1]
        w["views_bytes"] += float((members + sum(sz[:-1])) * d * es)
    total_flops = sum(w[k] for k in ("gemm_qkv", "gemm_o", "gemm_gateup",
                                     "gemm_down", "attention",
                                     "head_gemm_flops"))
    return w, total_flops


MATRIX_CLASSES = ("gemm_qkv", "gemm_o", "gemm_gateup", "gemm_down",
                  "attention")
ROOFLINE_CLASSES = MATRIX_CLASSES + ("head_gemm",)


def dominant_class(kern):
    """The kernel class (with an algorithmic-work model) that took the most
    time in a profiled pass."""
    ranked = sorted(((ms, name) for name, (cnt, ms) in kern.items()
                     if cnt and name in ROOFLINE_CLASSES), reverse=True)
    return ranked[0][1] if ranked else None


def measured_traffic(name, workload):
    """HBM bytes per launch of a kernel class, as measured by the FETCH_SIZE
    and WRITE_SIZE counters and scaled by a plain copy kernel's readings
    (profiles/<class>_<workload>.md).  None unless the kernel sources are
    byte-identical to those the counters were taken on."""
    import hashlib
    path = os.path.join(ROOT, "profiles", "%s_%s.md" % (name, workload))
    if not os.path.exists(path):
        return None
    fields = {}
    with open(path) as f:
        for line in f:
            if line.startswith("- ") and ": " in line:
                k, v = line[2:].strip().split(": ", 1)
                fields[k.strip("`")] = v.strip().strip("`")
    try:
        for src, want in zip(fields["sources"].split(","),
                             fields["sources_sha256"].split(",")):
            with open(os.path.join(ROOT, src.strip()), "rb") as f:
                if hashlib.sha256(f.read()).hexdigest()[:16] != want.strip():
                    return None
        return float(fields["traffic_bytes_per_launch"])
    except (KeyError, OSError, ValueError):
        return None


def roofline(cfg, name, cnt, ms, work, loops):
    """Roofline object of one kernel class from its timed launches."""
    if not name or cnt == 0:
        return None
    sec = ms / 1e3
    traffic = measured_traffic(name, cfg.name)
    if name in MATRIX_CLASSES:
        flops = work[name] * loops
        peak = PEAK_BF16_TFLOPS if cfg.dtype == "bf16" else PEAK_FP32_TFLOPS
        ach = flops / sec / 1e12
        return dict(kernel=name, bound="mfma", achieved=round(ach, 2),
                    peak=peak, unit="TFLOP/s", frac=round(ach / peak, 4),
                    traffic=traffic, traffic_unit="HBM bytes per launch",
                    launches=cnt, mean_launch_us=round(ms * 1e3 / cnt, 2))
    byts = work["head_gemm_bytes"] * loops
    ach = byts / sec / 1e9
    return dict(kernel=name, bound="hbm", achieved=round(ach, 1),
                peak=PEAK_HBM_GBS, unit="GB/s",
                frac=round(ach / PEAK_HBM_GBS, 4), traffic=traffic,
                traffic_unit="HBM bytes per launch",
                algorithmic_bytes_per_launch=round(byts / cnt),
                launches=cnt, mean_launch_us=round(ms * 1e3 / cnt, 2))


def kernel_rooflines(cfg, kern, work):
    """Every kernel class with a work model, from the untimed profiled pass
    (one loop): achieved rate and fraction of its roofline."""
    peak_mm = PEAK_BF16_TFLOPS if cfg.dtype == "bf16" else PEAK_FP32_TFLOPS
    out = {}
    for name, (cnt, ms) in kern.items():
        if not cnt or ms <= 0:
            continue
        sec = ms / 1e3
        if name in MATRIX_CLASSES:
            ach = work[name] / sec / 1e12
            out[name] = dict(bound="mfma", achieved=round(ach, 1),
                             unit="TFLOP/s", frac=round(ach / peak_mm, 4))
        elif name == "head_gemm":
            ach = work["head_gemm_bytes"] / sec / 1e9
            out[name] = dict(bound="hbm", achieved=round(ach, 1), unit="GB/s",
                             frac=round(ach / PEAK_HBM_GBS, 4))
        elif name in ("views", "realizer_keys"):
            ach = work[name + "_bytes"] / sec / 1e9
            out[name] = dict(bound="hbm", achieved=round(ach, 1), unit="GB/s",
                             frac=round(ach / PEAK_HBM_GBS, 4))
    return out


def per_level_steps(cfg, st, levels, reps=10, profile=True):
    """Denoising step time at every view level (the loop's own kernels, one
    davet_denoise_step + davet_unmask on every sequence at that level, all
    response positions masked), timed with events; untimed by the bench.
    With `profile`, one further step per level carries events around every
    launch and gives each matrix kernel class's rate at that level."""
    import torch
    dv = st["dv"]
    n, L, K = cfg.n_seqs, cfg.resp_len, cfg.K
    out = {}
    conf = torch.empty(n * L, device="cuda")
    am = torch.empty(n * L, dtype=torch.int32, device="cuda")
    for lv in range(K):
        views, nview = [], []
        for i in range(n):
            views.append(st["visual"][i] if lv == K - 1
                         else st["view_bufs"][i * (K - 1) + lv])
            nview.append(st["sizes"][i][lv])
        times = []
        for r in range(reps + 2):
            st["ids"].fill_(cfg.mask_id)
            st["msk"].fill_(1)
            e0 = torch.cuda.Event(enable_timing=True)
            e1 = torch.cuda.Event(enable_timing=True)
            e0.record()
            dv.davet_denoise_step(st["mcfg"], st["W"], views, nview,
                                  st["prompt"], st["cu"], st["ids"], st["msk"],
                                  L, conf, am, None, st["ws"])
            dv.davet_unmask(n, L, cfg.k, conf, am, st["ids"], st["msk"])
            e1.record()
            e1.synchronize()
            if r >= 2:
                times.append(e0.elapsed_time(e1))
        times.sort()
        ms = times[len(times) // 2]
        tokens = sum(nview) + st["cu"][-1] + n * L
        out[str(lv)] = dict(tokens=tokens, ms_per_step=round(ms, 4),
                            steps_per_s=round(1e3 / ms, 2))
        if profile and cfg.dtype == "bf16":
            # one more step with events around every launch: each matrix
            # class's rate at this level against the 2.5 PF peak
            st["ids"].fill_(cfg.mask_id)
            st["msk"].fill_(1)
            torch.cuda.synchronize()
            dv.prof_enable(12 * cfg.n_layers + 64)
            dv.davet_denoise_step(st["mcfg"], st["W"], views, nview,
                                  st["prompt"], st["cu"], st["ids"], st["msk"],
                                  L, conf, am, None, st["ws"])
            torch.cuda.synchronize()
            kern = dv.prof_read()
            dv.prof_enable(0)
            d, F = cfg.d, cfg.ffn
            lens = [nview[i] + st["cu"][i + 1] - st["cu"][i] + L
                    for i in range(n)]
            flops = {"gemm_qkv": 2.0 * tokens * d * 3 * d,
                     "gemm_o": 2.0 * tokens * d * d,
                     "gemm_gateup": 2.0 * tokens * d * 2 * F,
                     "gemm_down": 2.0 * tokens * F * d,
                     "attention": sum(4.0 * m * m * d for m in lens)}
            rates = {}
            for name, fl in flops.items():
                cnt, kms = kern.get(name, (0, 0.0))
                if cnt and kms > 0:
                    ach = cfg.n_layers * fl / (kms / 1e3) / 1e12
                    rates[name] = dict(achieved=round(ach, 1),
                                       frac=round(ach / PEAK_BF16_TFLOPS, 4))
            out[str(lv)]["matrix_rooflines_one_step"] = rates
    return out


def cpu_baseline(cfg, st, n_layers_run):
    """The oracle, as it stands, on this host: one step per level the
    schedule uses (all positions masked, first sample), weighted by how
    often the schedule uses each level.  The step is timed in its parts
    (embedding, the layers run, final norm + head), so that a stack deeper
    than the layers run is extrapolated by its per-layer time only."""
    import numpy as np
    from threadpoolctl import threadpool_info

    import synth
    from oracle import model, realizers, views

    levels = st["levels"]
    T = cfg.steps
    s0 = st["sample"]
    visual = synth.gen_visual(cfg, s0["n_crops"][:1])[0]
    if st.get("realizer", "pool") != "pool":
        lv_f, _ = realizers.build_views(visual, s0["n_crops"][0], cfg.grid,
                                        cfg.K, REALIZERS[st["realizer"]],
                                        cfg.dtype)
    else:
        lv_f, _ = views.build_views(visual, s0["n_crops"][0], cfg.grid, cfg.K,
                                    cfg.dtype, st.get("mixed_stride", 0))
    embed, head = synth.gen_embed(cfg), synth.gen_head(cfg)
    layers = [synth.gen_layer_weights(cfg, i) for i in range(n_layers_run)]
    L = cfg.resp_len
    resp = np.full(L, cfg.mask_id)
    masked = np.ones(L, np.uint8)
    used = sorted(set(levels[:T]))
    per_level, parts = {}, {}
    for lv in used:
        t0 = time.perf_counter()
        x = model.embed_sequence(lv_f[lv], s0["prompts"][0], resp, masked,
                                 embed, cfg.mask_id)
        ang = model.rope_angles(x.shape[0], cfg.head_dim, cfg.rope_theta)
        t1 = time.perf_counter()
        for w in layers:
            x = model.layer(x, w, cfg.n_heads, cfg.head_dim, cfg.rms_eps, ang)
        t2 = time.perf_counter()
        model.response_logits(x, L, masked, head, None, cfg.rms_eps)
        t3 = time.perf_counter()
        per_layer = (t2 - t1) / n_layers_run
        per_level[lv] = (t1 - t0) + per_layer * cfg.n_layers + (t3 - t2)
        parts[str(lv)] = dict(embed_s=round(t1 - t0, 3),
                              per_layer_s=round(per_layer, 3),
                              head_s=round(t3 - t2, 3))
    sec = sum(per_level[levels[t]] for t in range(T)) * cfg.n_seqs
    threads = 0
    for info in threadpool_info():
        if info.get("user_api") == "blas":
            threads = max(threads, info.get("num_threads", 0))
    extrap = n_layers_run < cfg.n_layers
    sample = ("one oracle step per level %s of sample 0 (all positions "
              "masked), float64 numpy, %d of %d layers run%s; weighted by the "
              "schedule's %d steps%s" % (
                  used, n_layers_run, cfg.n_layers,
                  " (extrapolated: embedding + %d x the measured per-layer "
                  "time + head)" % cfg.n_layers if extrap else "", T,
                  " x %d samples" % cfg.n_seqs if cfg.n_seqs > 1 else ""))
    return dict(value=round(T / sec, 5), unit="denoise steps/s",
                cores=threads or len(os.sched_getaffinity(0)), kind="oracle",
                sample=sample, extrapolated=extrap,
                seconds_per_level={str(k): round(v, 3)
                                   for k, v in per_level.items()},
                parts_per_level=parts)


def other_workload(cid, args):
    """A short measurement of another workload (same loop, same timing rule:
    one warm-up loop, then two timed loops; one untimed profiled loop for
    the dominant kernel class and its roofline)."""
    import gc

    import torch
    import synth

    cfg = synth.get_config(cid)
    mode = args.mode if cfg.dtype == "bf16" else "f32"
    st = setup(cfg, mode, args.head_layout)
    dv = st["dv"]
    run_loop(cfg, st)
    torch.cuda.synchronize()
    per_loop = cfg.steps * (12 * cfg.n_layers + 16) + 64
    dv.prof_enable(per_loop)
    levels, _ = run_loop(cfg, st)
    torch.cuda.synchronize()
    kern = dv.prof_read()
    dv.prof_enable(0)
    st["levels"] = levels
    work, flops_loop = work_per_loop(cfg, st, levels)
    dom = dominant_class(kern)
    reps = 2
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(reps):
        run_loop(cfg, st)
    torch.cuda.synchronize()
    el = time.perf_counter() - t0
    k_roof = kernel_rooflines(cfg, kern, work)
    out = dict(workload=cfg.name, value=round(reps * cfg.steps / el, 3),
               unit="denoise steps/s", loops_timed=reps,
               ms_per_denoise_step=round(el / reps / cfg.steps * 1e3, 4),
               tflops_algorithmic=round(flops_loop * reps / el / 1e12, 2),
               dominant_kernel=dom,
               dominant_roofline_untimed_pass=k_roof.get(dom),
               kernel_rooflines_untimed_pass=k_roof)
    del st
    gc.collect()
    torch.cuda.empty_cache()
    return out


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: this build has no multi-GPU "
              "path (requested --gpus %d, WORLD_SIZE %d)" % (args.gpus, world),
              file=sys.stderr)
        sys.exit(2)
    if args.copy_calibration:
        copy_calibration(args.copy_calibration)
        return
    if args.views_probe:
        views_probe()
        return
    import torch
    import synth

    cfg = synth.get_config(args.config)
    if args.schedule == "policy" and cfg.schedule != "policy":
        import dataclasses
        cfg = dataclasses.replace(cfg, schedule="policy")
    mode = args.mode if cfg.dtype == "bf16" else "f32"
    if args.mixed_stride and args.realizer != "pool":
        print("the mixed view is a pooling level: --mixed-stride needs "
              "--realizer pool", file=sys.stderr)
        sys.exit(2)
    st = setup(cfg, mode, args.head_layout, args.mixed_stride, args.realizer)
    dv = st["dv"]
    for _ in range(args.warmup):
        run_loop(cfg, st)
    torch.cuda.synchronize()

    # one untimed pass with events around every launch: the schedule taken,
    # the per-class breakdown and the dominant kernel class
    per_loop = cfg.steps * (12 * cfg.n_layers + 16) + 64
    if not args.no_kernel_timing:
        dv.prof_enable(per_loop)
    levels, _ = run_loop(cfg, st)
    torch.cuda.synchronize()
    kern = {}
    if not args.no_kernel_timing:
        kern = dv.prof_read()
        dv.prof_enable(0)
    st["levels"] = levels
    work, flops_loop = work_per_loop(cfg, st, levels)
    dom = dominant_class(kern)

    # timed region: events only around the dominant class's launches
    if dom:
        dv.prof_enable(args.steps * per_loop)
        dv.prof_only(dom)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(args.steps):
        run_loop(cfg, st)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    rl = None
    if dom:
        cnt, ms = dv.prof_read()[dom]
        dv.prof_only(None)
        dv.prof_enable(0)
        rl = roofline(cfg, dom, cnt, ms, work, args.steps)
    elapsed = t1 - t0
    loops = args.steps
    steps_per_s = loops * cfg.steps / elapsed
    ms_loop = elapsed / loops * 1e3

    kernels = {k: dict(launches=c, total_ms=round(ms, 3),
                       mean_us=round(ms * 1e3 / c, 2) if c else 0.0)
               for k, (c, ms) in kern.items() if c}
    k_roof = kernel_rooflines(cfg, kern, work) if kern else {}
    views_ms = sum(kern.get(k, (0, 0.0))[1] for k in (
        "views", "view_maps", "realizer_keys", "realizer_maps")) \
        if kern else None
    crossing = None
    if args.crossing and st["pols"] is not None:
        # the same levels as a fixed schedule: the difference per step is the
        # policy's handshake (signals + allocation on the GPU, levels to host)
        pols = st["pols"]
        st["pols"], st["fixed"] = None, list(levels)
        run_loop(cfg, st)
        torch.cuda.synchronize()
        f0 = time.perf_counter()
        for _ in range(args.steps):
            run_loop(cfg, st)
        torch.cuda.synchronize()
        fixed_ms = (time.perf_counter() - f0) / args.steps * 1e3
        st["pols"], st["fixed"] = pols, None
        crossing = dict(policy_ms_per_loop=round(ms_loop, 3),
                        same_levels_fixed_ms_per_loop=round(fixed_ms, 3),
                        us_per_step=round((ms_loop - fixed_ms) / cfg.steps
                                          * 1e3, 2),
                        share=round((ms_loop - fixed_ms) / ms_loop, 5))
    levels_probe = per_level_steps(cfg, st, levels,
                                   profile=not args.no_kernel_timing)
    cpu = None
    if not args.no_cpu_baseline:
        try:
            cpu = cpu_baseline(cfg, st, max(1, min(args.cpu_layers,
                                                   cfg.n_layers)))
        except Exception as e:  # report, never hide, a failed baseline
            cpu = dict(error=repr(e))
    hist = {}
    for lv in levels:
        hist[str(lv)] = hist.get(str(lv), 0) + 1
    out = {
        "metric": "denoise steps/s + %bf16-MFMA-peak, 8B-shaped stack, "
                  "729-3645 visual tokens",
        "value": round(steps_per_s, 3),
        "unit": "denoise steps/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_loop, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": mode,
        "data": "synthetic (seeded N(0,0.02) weights, N(0,1) visual "
                "encodings, uniform prompt ids)",
        "config": {
            "workload": cfg.name, "model_dtype": cfg.dtype,
            "head_layout": args.head_layout if cfg.dtype == "bf16" else "rows",
            "realizer": args.realizer,
            "middle_view": ("mixed, lattice stride %d" % args.mixed_stride
                            if args.mixed_stride else
                            {"pool": "pooled (2x2 windows)",
                             "prune": "pruned (top-n by L1 norm)",
                             "merge": "merged (single linkage)"}[
                                 args.realizer]),
            "operands": {"f16": "fp16 x fp16 -> fp32 matrix cores, bf16 "
                                "weights rounded to fp16 (exact for "
                                "|w| >= 2^-17)",
                         "bf16": "bf16 x bf16 -> fp32 matrix cores",
                         "f32": "fp32 vector ALU"}[mode],
            "n_layers": cfg.n_layers, "d": cfg.d, "heads": cfg.n_heads,
            "head_dim": cfg.head_dim, "ffn": cfg.ffn, "vocab": cfg.vocab,
            "visual_tokens": [sz[-1] for sz in st["sizes"]],
            "view_levels_tokens": st["sizes"][0],
            "prompt": [st["cu"][i + 1] - st["cu"][i]
                       for i in range(cfg.n_seqs)],
            "response": cfg.resp_len, "denoise_steps_per_step": cfg.steps,
            "commit_per_step": cfg.k, "n_seqs": cfg.n_seqs,
            "schedule": cfg.schedule, "level_histogram": hist,
            "parallelism": "none (one GPU)",
        },
        "ms_per_denoise_step": round(ms_loop / cfg.steps, 4),
        "tflops_algorithmic": round(flops_loop * loops / elapsed / 1e12, 2),
        "roofline": rl,
        "kernels_untimed_pass": kernels,
        "kernel_rooflines_untimed_pass": k_roof,
        "views_vs_loop": None if views_ms is None else dict(
            views_ms=round(views_ms, 4), loop_ms=round(ms_loop, 3),
            share=round(views_ms / ms_loop, 6)),
        "per_level_all_masked": levels_probe,
        "policy_crossing": crossing,
        "cpu_baseline": cpu,
        "other_workloads": None,
    }
    if mode == "bf16" and cfg.n_layers > 2:
        out["accuracy_note"] = (
            "bf16 operands: logits rel-RMS measured 2.2e-2 at 32 layers, "
            "outside the 1e-2 tolerance; the f16 mode is the validated one")
        log("warning: " + out["accuracy_note"])
    others = {}
    if args.also:
        del st, dv
        import gc
        gc.collect()
        torch.cuda.empty_cache()
        for cid in [int(x) for x in args.also.split(",") if x.strip()]:
            if cid == args.config:
                continue
            log("other workload: config %d" % cid)
            try:
                others[str(cid)] = other_workload(cid, args)
            except Exception as e:   # report, never hide, a failed run
                others[str(cid)] = dict(error=repr(e))
    out["other_workloads"] = others
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
