"""Throughput of one DiT block forward on one MI355X.

One step = one pass of the whole hot path over one batch: timestep
conditioning, modulated LayerNorm, QKV projection, QK-RMSNorm + rotary,
self-attention, gated output projection, cross-attention to text, gated GELU
MLP.  The default workload is the 720p video block (75,600 latent tokens,
D = 5120, 40 heads of 128, MLP 13824, 512 text tokens), bf16 with fp32
accumulation, seeded synthetic inputs resident in HBM before timing starts.

The timed step runs the block through the library's seam entry points
(pre-attention -> attention -> post-attention; bitwise equal to
dit_block_forward) so that HIP events on the library's stream bracket the
self-attention kernel, the dominant one, inside the timed region.  The
dit_block_forward entry point is timed as well.

Prints ONE JSON line (rank 0).  --gpus > 1 is refused: this build runs on one
GPU.
"""
import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "DiT block fwd ms + TFLOP/s (% bf16 MFMA peak) at 32K/75K video tokens"
PEAK_BF16_TFLOPS = 2500.0
PEAK_FP32_TFLOPS = 157.3
PEAK_HBM_GBS = 8000.0
PROFILE_TRAFFIC = os.path.join(ROOT, "profiles", "attn_fwd_bf16.video_720p.traffic.txt")
ATTN_SOURCE = os.path.join(ROOT, "paper_2606_13501_amd", "csrc", "attention.hip")



class GpuSensors:
    """Power and shader clock of the GPU while the timed steps run.

    A background thread reads sysfs every `period` seconds: the board power
    (`hwmon*/power1_input`, microwatts) and the current shader clock (the line
    of `pp_dpm_sclk` marked with `*`).  These are file reads only; no external
    tool is started.  On a box with several GPUs the first card that exposes
    the files is read.  Missing files give None."""

    def __init__(self, period=0.02, root="/sys/class/drm"):
        import glob
        cards = sorted(glob.glob(os.path.join(root, "card*", "device", "pp_dpm_sclk")))
        self.sclk = cards[0] if cards else None
        dev = os.path.dirname(self.sclk) if self.sclk else ""
        power = sorted(glob.glob(os.path.join(dev, "hwmon", "hwmon*", "power1_input"))) if dev else []
        self.power = power[0] if power else None
        self.cap = os.path.join(os.path.dirname(self.power), "power1_cap") if self.power else None
        self.period = period
        self.watts, self.mhz = [], []
        self._stop = None
        self._thread = None

    @staticmethod
    def _read(path):
        try:
            with open(path) as f:
                return f.read()
        except OSError:
            return None

    def _sample(self):
        if self.power:
            v = self._read(self.power)
            if v and v.strip().isdigit():
                self.watts.append(int(v) / 1e6)
        if self.sclk:
            v = self._read(self.sclk)
            for line in (v or "").splitlines():
                if line.rstrip().endswith("*"):
                    num = "".join(ch for ch in line.split(":", 1)[-1] if ch.isdigit())
                    if num:
                        self.mhz.append(int(num))

    def __enter__(self):
        import threading
        if self.power or self.sclk:
            self._stop = threading.Event()

            def loop():
                while not self._stop.is_set():
                    self._sample()
                    self._stop.wait(self.period)

            self._thread = threading.Thread(target=loop, daemon=True)
            self._thread.start()
        return self

    def __exit__(self, *exc):
        if self._thread is not None:
            self._stop.set()
            self._thread.join()
        return False

    def summary(self):
        cap = self._read(self.cap) if self.cap else None
        w, m = self.watts, sorted(self.mhz)
        return {
            "gpu_power_w_mean": round(sum(w) / len(w), 1) if w else None,
            "gpu_power_w_max": round(max(w), 1) if w else None,
            "gpu_power_cap_w": round(int(cap) / 1e6, 1) if cap and cap.strip().isdigit() else None,
            "gpu_sclk_mhz_median": m[len(m) // 2] if m else None,
            "gpu_sensor_samples": len(w),
        }

def block_flops(wl):
    """Algorithmic flops of one block (2 per multiply-add; attention 4 n^2 H d
    non-causal for self, 4 n L H d for cross)."""
    D, F, Dff, d = wl.hidden, wl.freq_dim, wl.mlp_hidden, wl.head_dim
    T, R, Lt = wl.n_rows, wl.n_req, wl.n_txt
    a_rows = wl.attn_rows if wl.attn_rows is not None else wl.rows
    a_heads = wl.attn_heads if wl.attn_heads is not None else wl.n_heads
    f = {
        "cond": 2.0 * R * (D * F + D * D + 6 * D * D),
        "gemm": 2.0 * T * D * (3 * D + D + D + D + 2 * Dff) + 2.0 * Lt * D * 2 * D,
        "self_attn": sum(4.0 * n * n * a_heads * d for n in a_rows),
        "cross_attn": sum(4.0 * n * wl.txt_len * wl.n_heads * d for n in wl.rows),
    }
    f["total"] = sum(f.values())
    return f


def read_traffic():
    """HBM bytes per attention launch from the committed rocprofv3 counter
    summary, or None when it is missing or was taken on another kernel source."""
    if not os.path.exists(PROFILE_TRAFFIC):
        return None
    kv = {}
    for line in open(PROFILE_TRAFFIC):
        if "=" in line and not line.lstrip().startswith("#"):
            k, v = line.split("=", 1)
            kv[k.strip()] = v.strip()
    src_sha = hashlib.sha256(open(ATTN_SOURCE, "rb").read()).hexdigest()[:16]
    if kv.get("kernel_source_sha256_16") != src_sha:
        return None
    try:
        return float(kv["traffic_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def cpu_baseline(wl, target_s=12.0):
    """The oracle (float64 NumPy) on a bounded sample of the same workload:
    every per-token step for n sampled query rows of the request, with their
    self-attention over all of the request's keys (seeded K and V, all heads)
    and cross-attention over its text.  Reported in TFLOP/s of the sample's
    algorithmic flops."""
    import numpy as np
    import synth
    from oracle import dit_block as O
    try:
        from threadpoolctl import threadpool_info
        cores = max([i.get("num_threads", 1) for i in threadpool_info() if i.get("user_api") == "blas"] or [1])
    except Exception:
        cores = len(os.sched_getaffinity(0))
    inp = synth.generate_block_inputs(wl)
    w = {k: O.decode(v) for k, v in inp.items()}
    del inp
    att = synth.generate_attention_inputs(wl)
    D, H, d = wl.hidden, wl.n_heads, wl.head_dim
    K = O.decode(att["k"]).reshape(-1, H * d)
    V = O.decode(att["v"]).reshape(-1, H * d)
    del att
    cfg = O.config_from_workload(wl)
    n_all = wl.rows[0]

    def run(n):
        rows = np.linspace(0, n_all - 1, n).astype(np.int64)
        t0 = time.perf_counter()
        mod = O.conditioning(w["t"], cfg.freq_dim, w)
        # per-token pre-attention steps on the sampled rows: each row is its own
        # one-row request at its grid position, all sharing the request's modulation
        rows_vl = O.Varlen(list(range(n + 1)), [0] * (n + 1), [wl.grids[0]] * n, [int(r) for r in rows])
        q, _, _ = O.pre_attention(cfg, rows_vl, w["x"][rows], w, np.broadcast_to(mod, (n,) + mod.shape[1:]))
        sub = O.Varlen([0, n], [0, wl.txt_len], [wl.grids[0]])
        o = O.attention_varlen(q, K, V, [0, n], [0, n_all], H, d)
        O.post_attention(cfg, sub, w["x"][rows], o, w["txt"], w, mod)
        dt = time.perf_counter() - t0
        Dff = wl.mlp_hidden
        fl = n * (2.0 * D * (3 * D + 3 * D + 2 * Dff) + 4.0 * n_all * H * d + 4.0 * wl.txt_len * H * d) \
            + 2.0 * wl.txt_len * D * 2 * D + 2.0 * (D * wl.freq_dim + 7 * D * D)
        return dt, fl

    # two probes give the fixed cost (conditioning, text projection) and the
    # cost per sampled row, so the sample lands near target_s
    n1, n2 = min(16, n_all), min(64, n_all)
    dt1, _ = run(n1)
    dt2, _ = run(n2)
    per_row = max((dt2 - dt1) / max(n2 - n1, 1), 1e-6)
    fixed = max(dt1 - n1 * per_row, 0.0)
    n = int(min(4096, n_all, max(n2, (target_s - fixed) / per_row)))
    dt, fl = run(n)
    return {"value": fl / dt / 1e12, "unit": "TFLOP/s", "cores": int(cores), "kind": "oracle",
            "sample": (f"{wl.name}: all block steps for {n} evenly spaced query rows of the "
                       f"{n_all}-token request (self-attention of those rows over all {n_all} keys, "
                       f"{H} heads, seeded K/V; cross-attention over {wl.txt_len} text tokens); "
                       f"float64 NumPy, {dt:.1f} s")}


STEP_METRIC = "DiT denoising step ms + TFLOP/s (% bf16 MFMA peak): B blocks + patch embedding + output layer + Euler"


def step_flops(mw):
    """Algorithmic flops of one denoising step: B blocks without their own
    timestep MLP and text key/value projection (shared and cached), plus the
    shared timestep MLP, the patch embedding, the output modulation and
    projection (the Euler update is 2 flops per latent value)."""
    wl = mw.block
    D, F, P, R = wl.hidden, wl.freq_dim, mw.patch_len, wl.n_req
    fb = block_flops(wl)
    per_block = fb["total"] - 2.0 * R * (D * F + D * D) - 2.0 * wl.n_txt * D * 2 * D
    head = 2.0 * R * (D * F + D * D) + 2.0 * wl.n_rows * P * D * 2 + 2.0 * R * 2 * D * D
    return {"blocks": mw.n_blocks * per_block, "self_attn": mw.n_blocks * fb["self_attn"],
            "total": mw.n_blocks * per_block + head + 2.0 * sum(mw.latent_sizes())}


def run_step(args):
    """Time dit_denoise_step at a step workload (weights drawn on the device:
    the block recipe's distributions from torch's seeded device generator, so
    that 40 blocks of weights need no host round trip)."""
    import torch
    import synth
    import paper_2606_13501_amd.binding as B
    mw = synth.get_model_workload(args.step)
    wl = mw.block
    D, F, P, Dff, d = wl.hidden, wl.freq_dim, mw.patch_len, wl.mlp_hidden, wl.head_dim
    tdt = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
    g = torch.Generator(device="cuda")
    g.manual_seed(13501)

    def normal(shape, std=1.0, mean=0.0, dtype=tdt):
        return (torch.randn(shape, generator=g, device="cuda") * std + mean).to(dtype)

    t0 = time.time()
    std = wl.linear_std
    model = {"w_t1": normal((D, F), std), "b_t1": normal((D,), 0.02), "w_t2": normal((D, D), std),
             "b_t2": normal((D,), 0.02), "w_pe": normal((D, P), std), "b_pe": normal((D,), 0.02),
             "w_hmod": normal((2 * D, D), std), "b_hmod": normal((2 * D,), 0.02), "w_out": normal((P, D), std),
             "b_out": normal((P,), 0.02)}
    shapes = {"w_ada": (6 * D, D), "b_ada": (6 * D,), "w_qkv": (3 * D, D), "b_qkv": (3 * D,), "g_q": (d,),
              "g_k": (d,), "w_o": (D, D), "b_o": (D,), "g_ca": (D,), "b_ca": (D,), "w_cq": (D, D), "b_cq": (D,),
              "w_ckv": (2 * D, D), "b_ckv": (2 * D,), "g_cq": (d,), "g_ck": (d,), "w_co": (D, D), "b_co": (D,),
              "w_up": (Dff, D), "b_up": (Dff,), "w_dn": (D, Dff), "b_dn": (D,)}
    blocks = []
    for _ in range(mw.n_blocks):
        blk = {}
        for n, shp in shapes.items():
            if n.startswith("g_"):
                blk[n] = normal(shp, 0.02, 1.0)
            else:
                blk[n] = normal(shp, std if len(shp) == 2 else 0.02)
        blocks.append(blk)
    latent = torch.randn((sum(mw.latent_sizes()),), generator=g, device="cuda")
    txt = normal((wl.n_txt, D))
    t = torch.rand((wl.n_req,), generator=g, device="cuda") * 1000.0
    dt = -0.01 - 0.04 * torch.rand((wl.n_req,), generator=g, device="cuda")
    torch.cuda.synchronize()
    print(f"[bench] drew {mw.name} weights on the device in {time.time() - t0:.1f} s", file=sys.stderr, flush=True)

    bc = B.BlockConfig(D, wl.n_heads, d, Dff, F, wl.rope_sections, tdt)
    cfg = B.ModelConfig(bc, mw.n_blocks, mw.in_channels, mw.patch)
    w = B.ModelWeights(model, [B.make_weights(b) for b in blocks])
    vl = B.Varlen(wl.cu_seqlens(), wl.cu_txt(), list(wl.grids))
    ws = torch.empty(B.denoise_workspace_size(cfg, vl), dtype=torch.uint8, device="cuda")
    kv = torch.empty(B.text_kv_elems(cfg, vl), dtype=tdt, device="cuda")
    stream = torch.cuda.current_stream()
    k0, k1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    k0.record(stream)
    B.text_kv(cfg, w, vl, txt, kv)
    k1.record(stream)
    lat = [latent, torch.empty_like(latent)]

    def one(i):
        B.denoise_step(cfg, w, vl, lat[i % 2], t, dt, kv, lat[(i + 1) % 2], ws)

    for i in range(args.warmup):
        one(i)
        torch.cuda.synchronize()
        print(f"[bench] warmup step {i} done", file=sys.stderr, flush=True)
    start, stop = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    with GpuSensors() as sensors:
        start.record(stream)
        for i in range(args.steps):
            one(args.warmup + i)
        stop.record(stream)
        torch.cuda.synchronize()
    ms = start.elapsed_time(stop) / args.steps
    if not torch.isfinite(lat[(args.warmup + args.steps) % 2]).all():
        raise RuntimeError("non-finite latent after the timed steps")
    fl = step_flops(mw)
    tflops = fl["total"] / (ms * 1e-3) / 1e12
    out = {
        "metric": STEP_METRIC,
        "value": round(tflops, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if wl.dtype == "bf16" else "f32",
        "data": "synthetic (seeded device draws; random-init weights of the block recipe's distributions)",
        "config": {
            "workload": mw.name, "blocks": mw.n_blocks, "tokens": wl.n_rows, "requests": wl.n_req, "hidden": D,
            "heads": wl.n_heads, "head_dim": d, "mlp_hidden": Dff, "text_tokens": wl.n_txt,
            "latent_channels": mw.in_channels, "patch": list(mw.patch), "step_flops": fl["total"],
            "pct_bf16_peak": round(100.0 * tflops / PEAK_BF16_TFLOPS, 2),
            "ms_text_kv_once_per_request": round(k0.elapsed_time(k1), 3),
            "ms_per_block": round(ms / mw.n_blocks, 3),
            **sensors.summary(),
        },
        "roofline": {
            "kernel": "whole step (per-kernel durations: rocprofv3 kernel statistics of this command)",
            "bound": "mfma",
            "achieved": round(tflops, 2),
            "peak": PEAK_BF16_TFLOPS,
            "unit": "TFLOP/s",
            "frac": round(tflops / PEAK_BF16_TFLOPS, 4),
            "traffic": None,
        },
    }
    if not args.no_cpu_baseline:
        t0 = time.time()
        out["cpu_baseline"] = cpu_baseline(wl)
        out["cpu_baseline"]["sample"] += " (the oracle's rate on one block's work; a step is B such blocks)"
        print(f"[bench] cpu baseline took {time.time() - t0:.1f} s", file=sys.stderr, flush=True)
    print(json.dumps(out), flush=True)


XGMI_LINK_GBS = 153.0   # one xGMI link, one direction (MI355X: 7 links per GPU, one to each peer)


def run_cost_table(args):
    """Latency of one denoising step per (request class, sequence-parallel
    degree): one GPU's share of a block, timed on this GPU (per-token stages on
    its ceil(n/d) rows with all heads, self-attention over all n rows with H/d
    heads, seeded operands), times the model's depth, plus a model of the two
    all-to-alls per block (q, k, v out and o back: 4 (n/d) D bf16 values per
    GPU, 1/d of it to each peer over its own link).  Prints one JSON line per
    entry and a final line with the whole table."""
    import torch
    import synth
    import paper_2606_13501_amd.binding as B
    g = torch.Generator(device="cuda")
    g.manual_seed(13501)
    stream = torch.cuda.current_stream()
    table = {}
    for model in ("video", "image"):
        D, H, hd, Dff, F, sec, n_blocks, L = synth.MODEL_SHAPES[model]
        classes = [c for c in synth.REQUEST_CLASSES.values() if c.model == model]
        n_max = max(c.tokens for c in classes)

        def normal(shape, std=1.0, mean=0.0):
            return (torch.randn(shape, generator=g, device="cuda") * std + mean).to(torch.bfloat16)

        shapes = {"w_t1": (D, F), "b_t1": (D,), "w_t2": (D, D), "b_t2": (D,), "w_ada": (6 * D, D), "b_ada": (6 * D,),
                  "w_qkv": (3 * D, D), "b_qkv": (3 * D,), "g_q": (hd,), "g_k": (hd,), "w_o": (D, D), "b_o": (D,),
                  "g_ca": (D,), "b_ca": (D,), "w_cq": (D, D), "b_cq": (D,), "w_ckv": (2 * D, D), "b_ckv": (2 * D,),
                  "g_cq": (hd,), "g_ck": (hd,), "w_co": (D, D), "b_co": (D,), "w_up": (Dff, D), "b_up": (Dff,),
                  "w_dn": (D, Dff), "b_dn": (D,)}
        wd = {n: normal(shp, 0.02, 1.0 if n.startswith("g_") else 0.0) for n, shp in shapes.items()}
        w = B.make_weights(wd)
        x = normal((n_max, D))
        txt = normal((L, D))
        t = torch.rand((1,), generator=g, device="cuda") * 1000.0
        cfg = B.BlockConfig(D, H, hd, Dff, F, sec, torch.bfloat16)
        for c in classes:
            for deg in synth.SP_DEGREES:
                wl = synth.share_workload(c, deg)
                T = wl.rows[0]
                vl = B.Varlen([0, T], [0, L], [c.grid])
                ws = torch.empty(B.block_workspace_size(cfg, vl), dtype=torch.uint8, device="cuda")
                mod = torch.empty((1, 6, D), dtype=torch.float32, device="cuda")
                qkv = torch.empty((3, T, D), dtype=torch.bfloat16, device="cuda")   # q, k, v planes
                o = torch.empty((T, D), dtype=torch.bfloat16, device="cuda")
                y = torch.empty((T, D), dtype=torch.bfloat16, device="cuda")
                xs = x[:T]
                if deg > 1:
                    Ha, n = H // deg, c.tokens
                    qkv_a = normal((3, n, Ha * hd))
                    o_a = torch.empty((n, Ha * hd), dtype=torch.bfloat16, device="cuda")
                    o_rows = normal((T, D))

                def share():
                    B.block_pre_attention(cfg, w, vl, xs, t, mod, qkv, ws)
                    if deg > 1:
                        B.attention_varlen(qkv_a[0], qkv_a[1], qkv_a[2], o_a, [0, c.tokens], [0, c.tokens], Ha, hd)
                    else:
                        B.attention_varlen(qkv[0], qkv[1], qkv[2], o, [0, T], [0, T], H, hd)
                    B.block_post_attention(cfg, w, vl, xs, o_rows if deg > 1 else o, txt, mod, y, ws)

                for _ in range(args.warmup):
                    share()
                evs = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
                       for _ in range(args.steps)]
                torch.cuda.synchronize()
                for a, b in evs:
                    a.record(stream)
                    share()
                    b.record(stream)
                torch.cuda.synchronize()
                ms = sorted(a.elapsed_time(b) for a, b in evs)
                comm = 0.0 if deg == 1 else 4.0 * T * D * 2 / deg / (XGMI_LINK_GBS * 1e9) * 1e3
                step_ms = n_blocks * (ms[len(ms) // 2] + comm)
                table[(c.name, deg)] = step_ms
                print(json.dumps({"cost_entry": c.name, "tokens": c.tokens, "degree": deg, "rows": T,
                                  "attn_heads": H // deg, "block_ms_median": round(ms[len(ms) // 2], 4),
                                  "block_ms_min": round(ms[0], 4), "comm_ms_model": round(comm, 4),
                                  "blocks": n_blocks, "step_ms": round(step_ms, 3)}), flush=True)
                del ws, qkv, o, y
                if deg > 1:
                    del qkv_a, o_a, o_rows
        del wd, w, x
        torch.cuda.empty_cache()
    print(json.dumps({"cost_table_step_ms": {f"{k[0]}@{k[1]}": round(v, 3) for k, v in table.items()},
                      "degrees": list(synth.SP_DEGREES), "steps": args.steps, "warmup": args.warmup}), flush=True)


SIM_POLICIES = [("FCFS-SP1", 0, 1), ("FCFS-SP8", 0, 8), ("SRTF-SP1", 1, 1), ("SRTF-SP8", 1, 8), ("EDF-bestfit", 2, 1)]


def run_simulate(args):
    """Replay seeded traces of the paper's two workloads (mixed, foreground
    burst) for the video and the image classes on 8 ranks under each policy,
    with step costs from the measured cost table, in the library's simulator;
    the simulator oracle replays the same traces beside it for its timing.
    Prints one JSON line per (model, workload) and one with the simulators'
    event rates."""
    import numpy as np
    import synth
    import paper_2606_13501_amd.binding as B
    from oracle import sim as S
    step_ms = synth.read_cost_table(os.path.join(ROOT, "profiles", "step_cost_table.md"))
    degrees = list(synth.SP_DEGREES)
    G = 8
    lib_ev = lib_s = ora_ev = ora_s = 0.0
    for model, duration, allowance_s in (("video", 3600.0, 5.0), ("image", 600.0, 1.0)):
        for kind in ("mixed", "burst"):
            tr = synth.make_trace(kind, model, step_ms, G, duration, args.load, seed=0)
            cost = synth.cost_matrix(step_ms, tr["classes"], degrees)
            arr = np.asarray(tr["arrival_us"], dtype=np.int64)
            dl = np.asarray(tr["deadline_us"], dtype=np.int64)
            line = {"simulate": f"{model}/{kind}", "ranks": G, "requests": len(arr), "load": args.load,
                    "duration_s": duration, "policies": {}}
            for name, pol, grp in SIM_POLICIES:
                t0 = time.perf_counter()
                r = B.simulate(G, degrees, cost, pol, grp, arr, tr["cls"], tr["n_steps"], dl)
                lib_s += time.perf_counter() - t0
                lib_ev += r["events"]
                if args.sim_oracle:
                    t0 = time.perf_counter()
                    ro = S.simulate(G, degrees, cost, pol, grp, tr["arrival_us"], tr["cls"], tr["n_steps"],
                                    tr["deadline_us"])
                    ora_s += time.perf_counter() - t0
                    ora_ev += ro["events"]
                    if ro["finish"] != r["finish"].tolist():
                        raise RuntimeError(f"simulator and oracle differ on {model}/{kind} {name}")
                lat = (r["finish"] - arr) / 1e6
                met = r["finish"] <= dl + int(allowance_s * 1e6)
                line["policies"][name] = {
                    "slo_attainment": round(float(met.mean()), 4),
                    "mean_latency_s": round(float(lat.mean()), 2),
                    "p99_latency_s": round(float(np.percentile(lat, 99)), 2),
                    "makespan_s": round(float(r["finish"].max()) / 1e6, 1),
                    "steps_per_degree": dict(zip([str(d) for d in degrees], r["dispatches"].tolist())),
                }
            print(json.dumps(line), flush=True)
    rates = {"simulator_events_per_s": round(lib_ev / lib_s), "events": int(lib_ev)}
    if args.sim_oracle:
        rates["oracle_events_per_s"] = round(ora_ev / ora_s)
        rates["speedup"] = round((lib_ev / lib_s) / (ora_ev / ora_s), 1)
    print(json.dumps(rates), flush=True)


def run_migrate(args):
    """Rebuild the 720p video latent (fp32, channel-major 16 x 21 x 90 x 160,
    sharded by token rows, i.e. along its height in bands of whole token rows)
    from one sequence-parallel degree to another with the migration planner,
    executing the plan on this GPU (device buffers stand in for the ranks).
    Prints, per degree pair, the plan's entries and bytes, the device time of
    the execution and a model of the same transfers over xGMI (each entry one
    point-to-point transfer; a rank's sends share its link to the peer)."""
    import torch
    import paper_2606_13501_amd.binding as B
    from collections import defaultdict
    C, FL, HL, WL, ph = 16, 21, 90, 160, 2
    H = HL // ph
    g = torch.randn(C, FL, HL, WL, device="cuda")
    stream = torch.cuda.current_stream()

    def layout(d, base):
        # rank i owns token rows (f, h) with f*H + h in its ceil-split of F*H: here, h bands per frame
        # collapse to bands of the height that cover whole token rows, for every frame at once
        out = []
        for i in range(d):
            a, b = -(-H * i // d), -(-H * (i + 1) // d)
            out.append((base + i, [0, 0, a * ph, 0], [C, FL, b * ph, WL]))
        return out

    for d1 in (1, 2, 4, 8):
        for d2 in (1, 2, 4, 8):
            if d1 == d2:
                continue
            src, dst = layout(d1, 0), layout(d2, 16)
            f = B.MigField(B.MIG_SHARDED, (C, FL, HL, WL), 4, src, dst)
            entries, n = B.migration_plan(f)
            sb = [g[:, :, s[2]:e[2], :].contiguous() for _, s, e in src]
            db = [torch.empty(C, FL, e[2] - s[2], WL, device="cuda") for _, s, e in dst]
            for _ in range(args.warmup):
                B.migration_execute(f, entries, n, sb, db)
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            torch.cuda.synchronize()
            a.record(stream)
            for _ in range(args.steps):
                B.migration_execute(f, entries, n, sb, db)
            b.record(stream)
            torch.cuda.synchronize()
            ms = a.elapsed_time(b) / args.steps
            moved = sum(entries[k].bytes for k in range(n))
            remote = defaultdict(int)
            for k in range(n):
                if entries[k].src_rank != entries[k].dst_rank:
                    remote[(entries[k].src_rank, entries[k].dst_rank)] += entries[k].bytes
            xgmi_ms = max(remote.values()) / (XGMI_LINK_GBS * 1e9) * 1e3 if remote else 0.0
            print(json.dumps({"migrate": f"sp{d1}->sp{d2}", "entries": n, "bytes": moved,
                              "device_ms": round(ms, 4), "device_GBps": round(2 * moved / ms / 1e6, 1),
                              "xgmi_model_ms": round(xgmi_ms, 4)}), flush=True)
            for t in sb + db:
                del t


def profile_kernel(args, wl):
    """One kernel alone, args.steps times, for counter collection."""
    import torch
    import paper_2606_13501_amd.binding as B
    if args.profile_kernel == "copy":
        n = 1 << 29                                  # 2^29 two-byte elements = 1 GiB
        a = torch.empty(n, dtype=torch.float16, device="cuda").fill_(1.0)
        b = torch.empty_like(a)
        for _ in range(args.steps):
            b.copy_(a)
        torch.cuda.synchronize()
        print(json.dumps({"profile": "copy", "bytes_read": 2 * n, "bytes_written": 2 * n}), flush=True)
        return
    T, D, H, hd = wl.n_rows, wl.hidden, wl.n_heads, wl.head_dim
    g = torch.Generator(device="cuda")
    g.manual_seed(13501)
    if args.profile_kernel == "gated_residual":
        # the unfused gated residual (the block fuses it into the GEMM
        # epilogues): y = x + gate * (z + bias), timed with HIP events
        x = torch.randn((T, D), generator=g, device="cuda").to(torch.bfloat16)
        z = torch.randn((T, D), generator=g, device="cuda").to(torch.bfloat16)
        bias = (torch.randn((D,), generator=g, device="cuda") * 0.02).to(torch.bfloat16)
        gate = torch.randn((wl.n_req, D), generator=g, device="cuda")
        y = torch.empty_like(x)
        cu = wl.cu_seqlens()
        for _ in range(2):
            B.gated_residual(x, z, bias, gate, D, cu, y)
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        a.record()
        for _ in range(args.steps):
            B.gated_residual(x, z, bias, gate, D, cu, y)
        b.record()
        torch.cuda.synchronize()
        ms = a.elapsed_time(b) / args.steps
        alg = 3 * 2 * T * D   # x and z read, y written, once
        print(json.dumps({"profile": "gated_residual", "workload": wl.name, "launches": args.steps,
                          "ms_per_launch": round(ms, 4), "algorithmic_bytes": alg,
                          "achieved_gbs": round(alg / (ms * 1e-3) / 1e9, 1),
                          "frac_of_hbm_peak": round(alg / (ms * 1e-3) / 1e9 / PEAK_HBM_GBS, 4)}), flush=True)
        return
    qkv = torch.randn((3, T, D), generator=g, device="cuda").to(torch.bfloat16)   # q, k, v planes
    o = torch.empty((T, D), dtype=torch.bfloat16, device="cuda")
    cu = wl.cu_seqlens()
    for _ in range(args.steps):
        B.attention_varlen(qkv[0], qkv[1], qkv[2], o, cu, cu, H, hd)
    torch.cuda.synchronize()
    print(json.dumps({"profile": "attention", "workload": wl.name, "launches": args.steps}), flush=True)


def oracle_seconds(wl):
    """The float64 oracle on the workload's whole block, as it stands, on the
    host cores, timed by stages: conditioning and pre-attention on the rows,
    self-attention one (request, head) at a time with the oracle's attention
    (the loop its varlen attention runs, here with a progress line per head),
    post-attention on the rows.  For a sequence-parallel share the
    self-attention runs over the full lengths with the share's heads on the
    seeded q, k, v, and post-attention on the seeded attention output of the
    share's rows.  Prints seconds and fp64 GFLOP/s of the block's algorithmic
    work."""
    import numpy as np
    import synth
    from oracle import dit_block as O
    try:
        from threadpoolctl import threadpool_info
        blas = [i for i in threadpool_info() if i.get("user_api") == "blas"]
        cores = max([i.get("num_threads", 1) for i in blas] or [1])
        vendor = ",".join(sorted({i.get("internal_api", "?") for i in blas}))
    except Exception:
        cores, vendor = len(os.sched_getaffinity(0)), "?"
    inp = synth.generate_block_inputs(wl)
    w = {k: O.decode(v) for k, v in inp.items()}
    del inp
    cfg = O.config_from_workload(wl)
    vl = O.varlen_from_workload(wl)
    d = wl.head_dim
    stages = {}

    def note(msg):
        print(f"[oracle] {wl.name}: {msg}", file=sys.stderr, flush=True)

    t0 = time.perf_counter()
    mod = O.conditioning(w["t"], cfg.freq_dim, w)
    q, k, v = O.pre_attention(cfg, vl, w["x"], w, mod)
    stages["conditioning+pre_attention"] = time.perf_counter() - t0
    note(f"pre-attention {stages['conditioning+pre_attention']:.1f} s")
    if wl.is_sp_share:
        att = synth.generate_attention_inputs(wl)
        Ha = wl.attn_heads
        q, k, v = (O.decode(att[n]).reshape(-1, Ha * d) for n in ("q", "k", "v"))
        o_rows = O.decode(att["o"])
        cu_a = wl.cu_attn()
    else:
        Ha, cu_a = wl.n_heads, wl.cu_seqlens()
    o = np.zeros_like(q)
    t1 = time.perf_counter()
    for r in range(len(cu_a) - 1):
        a, b = cu_a[r], cu_a[r + 1]
        for h in range(Ha):
            cs = slice(h * d, (h + 1) * d)
            o[a:b, cs] = O.attention(q[a:b, cs], k[a:b, cs], v[a:b, cs], 1.0 / np.sqrt(d))
            note(f"self-attention request {r} head {h}: {time.perf_counter() - t1:.1f} s")
    stages["self_attention"] = time.perf_counter() - t1
    t2 = time.perf_counter()
    O.post_attention(cfg, vl, w["x"], o_rows if wl.is_sp_share else o, w["txt"], w, mod)
    stages["post_attention"] = time.perf_counter() - t2
    note(f"post-attention {stages['post_attention']:.1f} s")
    sec = sum(stages.values())
    fl = block_flops(wl)["total"]
    print(json.dumps({"oracle_seconds": round(sec, 2), "workload": wl.name, "stages_s": {k: round(v, 2) for k, v in
                      stages.items()}, "gflops_fp64": round(fl / sec / 1e9, 2), "block_flops": fl,
                      "blas_threads": int(cores), "blas": vendor, "cpu_count": os.cpu_count(),
                      "affinity": len(os.sched_getaffinity(0))}), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="video_720p")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--profile-kernel", choices=["attention", "copy", "gated_residual"], default=None,
                    help="run only one kernel (for rocprofv3 counter passes) and exit: the block's "
                         "self-attention at the workload's shape, a plain 1 GiB device copy used to "
                         "calibrate the HBM byte counters, or the unfused gated residual at the "
                         "workload's shape (timed; prints GB/s)")
    ap.add_argument("--step", default=None, metavar="STEP_WORKLOAD",
                    help="time one whole denoising step (dit_denoise_step) at this step workload, e.g. "
                         "step_video_720p, instead of the block; prints its own JSON line")
    ap.add_argument("--cold", action="store_true",
                    help="also time steps with a 1 GiB scratch write before each (inputs evicted from the caches)")
    ap.add_argument("--oracle-seconds", action="store_true",
                    help="only time the float64 oracle on the workload's whole block (by stages for a "
                         "sequence-parallel share) on the host cores and print one JSON line; no GPU needed")
    ap.add_argument("--cost-table", action="store_true",
                    help="measure the denoising-step cost table (request class x sequence-parallel degree) "
                         "from one GPU's share of a block and print it")
    ap.add_argument("--simulate", action="store_true",
                    help="replay seeded traces under each scheduling policy with the measured cost table "
                         "(CPU only) and print the policies' SLO attainment and latency")
    ap.add_argument("--sim-oracle", action="store_true", help="with --simulate: also time the simulator oracle")
    ap.add_argument("--load", type=float, default=0.8, help="with --simulate: offered load (fraction of capacity)")
    ap.add_argument("--migrate", action="store_true",
                    help="time the latent's migration between sequence-parallel layouts (plan + one-GPU execution)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py: this build runs on one GPU only (asked for --gpus {args.gpus}); "
              f"multi-GPU sharding is designed but not built", file=sys.stderr)
        sys.exit(2)

    if args.simulate:
        run_simulate(args)
        return
    if args.oracle_seconds:
        import synth
        oracle_seconds(synth.get_workload(args.workload))
        return

    import numpy as np
    import torch
    import synth
    import paper_2606_13501_amd.binding as B

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    B.lib()
    torch.cuda.set_device(0)
    if args.step:
        run_step(args)
        return
    if args.cost_table:
        run_cost_table(args)
        return
    if args.migrate:
        run_migrate(args)
        return
    wl = synth.get_workload(args.workload)
    if args.profile_kernel:
        profile_kernel(args, wl)
        return
    t0 = time.time()
    inp = synth.generate_block_inputs(wl)
    print(f"[bench] generated {wl.name} inputs in {time.time() - t0:.1f} s", file=sys.stderr, flush=True)

    def dev(a):
        if a.dtype == np.uint16:
            return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).cuda()
        return torch.from_numpy(a).cuda()

    d = {k: dev(v) for k, v in inp.items()}
    del inp
    tdt = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
    cfg = B.BlockConfig(wl.hidden, wl.n_heads, wl.head_dim, wl.mlp_hidden, wl.freq_dim, wl.rope_sections, tdt)
    w = B.make_weights(d)
    vl = B.Varlen(wl.cu_seqlens(), wl.cu_txt(), list(wl.grids))
    ws = torch.empty(B.block_workspace_size(cfg, vl), dtype=torch.uint8, device="cuda")
    T, D, H, hd = wl.n_rows, wl.hidden, wl.n_heads, wl.head_dim
    y = torch.empty_like(d["x"])
    mod = torch.empty((wl.n_req, 6, D), dtype=torch.float32, device="cuda")
    qkv = torch.empty((3, T, D), dtype=tdt, device="cuda")   # q, k, v planes, as pre-attention writes them
    o = torch.empty((T, D), dtype=tdt, device="cuda")
    cu = wl.cu_seqlens()
    stream = torch.cuda.current_stream()
    sp = wl.is_sp_share
    if sp:
        # one GPU's share of sequence parallelism: self-attention over the full
        # request lengths with the GPU's head slice (seeded q, k, v, as the
        # all-to-all would deliver them); the rows' attention output for the
        # post-attention steps is seeded too (the exchange back is not one GPU's work)
        g = torch.Generator(device="cuda")
        g.manual_seed(13501)
        Ha, cu_a = wl.attn_heads, wl.cu_attn()
        qkv_a = torch.randn((3, cu_a[-1], Ha * hd), generator=g, device="cuda").to(tdt)
        o_a = torch.empty((cu_a[-1], Ha * hd), dtype=tdt, device="cuda")
        o_rows = torch.randn((T, D), generator=g, device="cuda").to(tdt)

    def step(ev=None):
        B.block_pre_attention(cfg, w, vl, d["x"], d["t"], mod, qkv, ws)
        if ev is not None:
            ev[0].record(stream)
        if sp:
            B.attention_varlen(qkv_a[0], qkv_a[1], qkv_a[2], o_a, cu_a, cu_a, Ha, hd)
        else:
            B.attention_varlen(qkv[0], qkv[1], qkv[2], o, cu, cu, H, hd)
        if ev is not None:
            ev[1].record(stream)
        B.block_post_attention(cfg, w, vl, d["x"], o_rows if sp else o, d["txt"], mod, y, ws)

    def new_ev():
        return torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    evs = [new_ev() for _ in range(args.steps)]
    sevs = [new_ev() for _ in range(args.steps)]
    start, stop = new_ev()
    torch.cuda.synchronize()
    with GpuSensors() as sensors:
        start.record(stream)
        for i in range(args.steps):
            sevs[i][0].record(stream)
            step(evs[i])
            sevs[i][1].record(stream)
        stop.record(stream)
        torch.cuda.synchronize()
    ms = start.elapsed_time(stop) / args.steps
    attn_ms = sum(a.elapsed_time(b) for a, b in evs) / args.steps
    step_ms = sorted(a.elapsed_time(b) for a, b in sevs)

    # cold: a 1 GiB scratch write between steps evicts the inputs from the caches
    cold = None
    if args.cold:
        scratch = torch.empty(1 << 30, dtype=torch.uint8, device="cuda")
        cevs = [new_ev() for _ in range(args.steps)]
        for i in range(args.steps):
            scratch.fill_(i & 0xFF)
            cevs[i][0].record(stream)
            step()
            cevs[i][1].record(stream)
        torch.cuda.synchronize()
        cold = sorted(a.elapsed_time(b) for a, b in cevs)
        del scratch

    # the single-call entry point, same work (not for a sequence-parallel share,
    # whose attention spans rows that are not this GPU's)
    fwd_ms = None
    if not sp:
        fstart, fstop = new_ev()
        torch.cuda.synchronize()
        fstart.record(stream)
        for _ in range(args.steps):
            B.block_forward(cfg, w, vl, d["x"], d["t"], d["txt"], y, ws)
        fstop.record(stream)
        torch.cuda.synchronize()
        fwd_ms = fstart.elapsed_time(fstop) / args.steps

    fl = block_flops(wl)
    tflops = fl["total"] / (ms * 1e-3) / 1e12
    attn_flops = fl["self_attn"]
    attn_tflops = attn_flops / (attn_ms * 1e-3) / 1e12
    traffic = read_traffic() if wl.name == "video_720p" else None   # counters were taken at 720p
    peak = PEAK_BF16_TFLOPS if wl.dtype == "bf16" else PEAK_FP32_TFLOPS
    out = {
        "metric": METRIC,
        "value": round(tflops, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if wl.dtype == "bf16" else "f32",
        "data": f"synthetic (seeded; {wl.description}; random-init weights)",
        "config": {
            "workload": wl.name, "tokens": T, "requests": wl.n_req, "hidden": D, "heads": H, "head_dim": hd,
            "mlp_hidden": wl.mlp_hidden, "text_tokens": wl.n_txt, "rope_sections": list(wl.rope_sections),
            "block_flops": fl["total"], "pct_bf16_peak": round(100.0 * tflops / PEAK_BF16_TFLOPS, 2),
            "ms_per_step_block_forward_entry": round(fwd_ms, 3) if fwd_ms is not None else None,
            "ms_step_median": round(step_ms[len(step_ms) // 2], 3), "ms_step_min": round(step_ms[0], 3),
            "ms_step_cold_median": round(cold[len(cold) // 2], 3) if cold else None,
            "ms_step_cold_min": round(cold[0], 3) if cold else None,
            **sensors.summary(),
        },
        "roofline": {
            "kernel": "attn_fwd_bf16 (self-attention)" if wl.dtype == "bf16" else "attn_fwd_f32 (self-attention)",
            "bound": "mfma",
            "achieved": round(attn_tflops, 2),
            "peak": peak,
            "unit": "TFLOP/s",
            "frac": round(attn_tflops / peak, 4),
            "traffic": traffic,
            "flops_per_launch": attn_flops,
            "ms_per_launch": round(attn_ms, 3),
        },
    }
    if not args.no_cpu_baseline and not sp:   # a share's oracle timing: --oracle-seconds (by stages)
        t0 = time.time()
        out["cpu_baseline"] = cpu_baseline(wl)
        print(f"[bench] cpu baseline took {time.time() - t0:.1f} s", file=sys.stderr, flush=True)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
