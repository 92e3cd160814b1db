"""Benchmark of one VSD EM step (sample -> score -> backward) on one MI355X.

    python bench.py [--steps K] [--warmup W] [--config C3] [--no-cpu-baseline]

Workload (default): the LLaMA-3-8B / EAGLE-3-shaped batch, B=4 T=512 N=8 L=6,
target vocabulary 128256, draft vocabulary 32000 with a draft->target map,
bf16 logits already resident in HBM, synthetic and seeded.  One step = every
row of the batch through vsd_sample_score_paths (E-step draws and path
scoring in one pass over the logits) and vsd_weighted_loss_bwd on one stream.
The same step through the three separate calls (vsd_sample_paths,
vsd_score_paths, vsd_weighted_loss_bwd) is timed too and reported beside it,
and the step once more, both ways, with the top-K renormalised KL term on
(K = 10, "kl_variant"), and with exact context ("exact_context": each family
on its own rows, drawn depth by depth); "verification" times the decode-time
verification of the step's draft paths (vsd_verify_paths) and reports its
mean accepted length beside the mean expected accepted length.
W untimed steps, then exactly K steps timed between stream synchronisations;
per-call durations come from HIP events recorded on the stream the kernels
run on.

Prints one JSON line: value = path-tokens (live rows) per second of whole
steps; roofline = the dominant kernel against its bound (algorithmic bytes:
each live row's draft and target logits read once); cpu_baseline = the CPU
oracle timed on a bounded sample of the same workload (computed before the GPU
is touched, in worker processes).  The line also carries "fused_lm_head": the
same step in the fused LM-head variant on its own workload (B=2 T=512 N=8 L=6,
hidden 4096, LM-head weights 128256 x 4096 and 32000 x 4096 bf16), against the
bf16 matrix-core peak.  --config C5 makes that workload the line's own.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, GB/s
# VALU issue peak without packed fp32: 256 CUs x 4 SIMDs x 16 lanes x 2.4 GHz
# (a wave64 instruction occupies a SIMD for 4 cycles), in lane-ops per second
VALU_PEAK_TOPS = 256 * 4 * 16 * 2.4e9 / 1e12
MFMA_BF16_PEAK_TFLOPS = 2500.0  # MI355X dense bf16 matrix-core peak, TFLOP/s

METRIC = "path-tokens scored/sec (fwd+bwd) and achieved HBM GB/s at V=128256"


_SAMPLE = None  # (X, Y, d2t, N, L) shared with forked workers


def _oracle_position(k):
    """Position k of the sample through the CPU oracle (worker process)."""
    from oracle import reference
    X, Y, d2t, N, L = _SAMPLE
    per = N * L
    t0 = time.perf_counter()
    reference.run_positions(X[k * per:(k + 1) * per], Y[k * per:(k + 1) * per], d2t, None, [k], N, L, {},
                            seed=0, offset=0)
    return time.perf_counter() - t0


def cpu_baseline(cfg, workers, per_worker=8):
    """Time the oracle on workers*per_worker positions of the workload, the
    positions spread over `workers` forked processes."""
    global _SAMPLE
    import multiprocessing as mp

    from synth import make_inputs, scaled
    # a CPU-generated sample of the same recipe (the GPU is not touched here)
    npos = workers * per_worker
    sample_cfg = scaled(cfg.name, name=cfg.name + "-cpu-sample", B=1, T=npos)
    inp = make_inputs(sample_cfg, "cpu", chunk_rows=1024)
    X = inp["X"][:, :cfg.v_draft].float().numpy()
    Y = inp["Y"][:, :cfg.v_target].float().numpy()
    d2t = None if inp["d2t"] is None else inp["d2t"].numpy()
    del inp
    _SAMPLE = (X, Y, d2t, cfg.N, cfg.L)
    t0 = time.perf_counter()
    with mp.get_context("fork").Pool(workers) as pool:
        pool.map(_oracle_position, range(npos), chunksize=per_worker)
    wall = time.perf_counter() - t0
    _SAMPLE = None
    rows = npos * cfg.N * cfg.L
    return {"value": rows / wall, "unit": "path-tokens/s", "cores": workers, "kind": "oracle",
            "sample": f"{npos} positions ({rows} path-tokens) of the {cfg.name} recipe, sample+score+grad, "
                      f"{workers} worker processes, {wall:.1f} s wall", **host_cpu_info()}


def _oracle_lm_position(k):
    """Position k of the LM-head sample through the CPU oracle (worker process)."""
    from oracle import lmhead
    Hd, Ht, Wd, Wt, d2t, N, L = _SAMPLE
    per = N * L
    t0 = time.perf_counter()
    lmhead.run_positions(Hd[k * per:(k + 1) * per], Ht[k * per:(k + 1) * per], Wd, Wt, d2t, None, [k], N, L, {},
                         seed=0, offset=0)
    return time.perf_counter() - t0


def cpu_baseline_lm(cfg, workers, per_worker=1):
    """The LM-head oracle (float64 logits, then the per-position oracle) on
    workers*per_worker positions of the fused workload."""
    global _SAMPLE
    import multiprocessing as mp

    from synth import make_inputs, scaled
    npos = workers * per_worker
    sample_cfg = scaled(cfg.name, name=cfg.name + "-cpu-sample", B=1, T=npos)
    inp = make_inputs(sample_cfg, "cpu")
    f32 = lambda t: t.float().numpy()
    _SAMPLE = (f32(inp["Hd"]), f32(inp["Ht"]), f32(inp["Wd"]), f32(inp["Wt"]), inp["d2t"].numpy(), cfg.N, cfg.L)
    del inp
    t0 = time.perf_counter()
    with mp.get_context("fork").Pool(workers) as pool:
        pool.map(_oracle_lm_position, range(npos), chunksize=per_worker)
    wall = time.perf_counter() - t0
    _SAMPLE = None
    rows = npos * cfg.N * cfg.L
    return {"value": rows / wall, "unit": "path-tokens/s", "cores": workers, "kind": "oracle",
            "sample": f"{npos} positions ({rows} path-tokens) of the {cfg.name} recipe, float64 LM-head logits + "
                      f"sample+score+grad, {workers} worker processes, {wall:.1f} s wall", **host_cpu_info()}


def host_cpu_info():
    """The host's logical CPU count, the CPUs this process may run on and the
    CPU model (from /proc/cpuinfo)."""
    model = None
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    model = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    try:
        usable = len(os.sched_getaffinity(0))
    except (AttributeError, OSError):
        usable = None
    return {"host_cpus": os.cpu_count(), "usable_cpus": usable, "cpu_model": model}


def default_workers():
    """Worker processes of the oracle timing: the CPUs this process may use,
    at most 16 (one GPU's share of the host)."""
    info = host_cpu_info()
    return max(1, min(16, info["usable_cpus"] or info["host_cpus"] or 1))


def copy_calibration(mib, dev):
    """One plain device copy of `mib` MiB: the PMC byte counters of this
    dispatch calibrate those of the kernels."""
    import torch
    src_buf = torch.ones(mib << 20, dtype=torch.uint8, device=dev)
    dst_buf = torch.empty_like(src_buf)
    torch.cuda.synchronize()
    dst_buf.copy_(src_buf)
    torch.cuda.synchronize()
    del src_buf, dst_buf


def bench_lm_head(cfg, steps, warmup, dev):
    """One EM step of the fused LM-head variant: vsd_sample_score_paths and
    vsd_weighted_loss_bwd on LmHead sources.  Returns timings and the
    matrix-core roofline of the forward (the dominant kernel)."""
    import torch

    import paper_2602_05774_amd as vsd
    from synth import make_inputs
    t0 = time.perf_counter()
    inp = make_inputs(cfg, dev)
    torch.cuda.synchronize()
    print(f"[bench] inputs {cfg.name} generated in {time.perf_counter() - t0:.1f} s", flush=True)
    prob = vsd.Problem(cfg.B, cfg.T, cfg.N, cfg.L, cfg.v_draft, cfg.v_target)
    params = vsd.Params(temp_draft=cfg.temp_draft, temp_target=cfg.temp_target)
    Xs, Ys = vsd.LmHead(inp["Hd"], inp["Wd"]), vsd.LmHead(inp["Ht"], inp["Wt"])
    out = vsd.alloc_score_outputs(prob, dev)
    ws = torch.empty(vsd.score_workspace_bytes(prob, torch.bfloat16, cfg.hidden), dtype=torch.uint8, device=dev)
    tok = [torch.empty(prob.R, dtype=torch.int32, device=dev) for _ in range(3)]
    grad = vsd.LmHeadGrad(torch.empty(prob.R, cfg.hidden, dtype=torch.bfloat16, device=dev),
                          torch.empty(prob.R, (cfg.v_draft + 7) // 8 * 8, dtype=torch.bfloat16, device=dev))
    err = torch.zeros(1, dtype=torch.int32, device=dev)

    def step(ev=None):
        if ev:
            ev[0].record()
        vsd.sample_score_paths(prob, params, Xs, Ys, inp["d2t"], inp["valid_depth"], cfg.philox_seed,
                               cfg.philox_offset, out=out, workspace=ws, tokens=tok)
        if ev:
            ev[1].record()
        vsd.weighted_loss_bwd(prob, params, Xs, out.lse_draft, tok[0], tok[1], out.coef_a, out.coef_b, grad=grad,
                              device_error=err)
        if ev:
            ev[2].record()

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(3)] for _ in range(steps)]
    t0 = time.perf_counter()
    for k in range(steps):
        step(evs[k])
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    t_fwd = sum(e[0].elapsed_time(e[1]) for e in evs) / steps
    t_bwd = sum(e[1].elapsed_time(e[2]) for e in evs) / steps
    # the backward once more with the draft weight's gradient (g^T H_d, fp32)
    gw = vsd.LmHeadGrad(grad.grad_hidden, grad.grad_logits,
                        torch.empty(cfg.v_draft, cfg.hidden, dtype=torch.float32, device=dev))
    ew = [torch.cuda.Event(enable_timing=True) for _ in range(2)]
    vsd.weighted_loss_bwd(prob, params, Xs, out.lse_draft, tok[0], tok[1], out.coef_a, out.coef_b, grad=gw,
                          device_error=err)
    ew[0].record()
    vsd.weighted_loss_bwd(prob, params, Xs, out.lse_draft, tok[0], tok[1], out.coef_a, out.coef_b, grad=gw,
                          device_error=err)
    ew[1].record()
    torch.cuda.synchronize()
    t_bwd_w = ew[0].elapsed_time(ew[1])
    del gw
    # the step once more with the top-K renormalised KL term (K = 10)
    params_kl = vsd.Params(temp_draft=cfg.temp_draft, temp_target=cfg.temp_target, kl_weight=0.1, kl_topk=10)
    out_kl = vsd.alloc_score_outputs(prob, dev, kl_topk=10)
    ek = [torch.cuda.Event(enable_timing=True) for _ in range(3)]
    for rep in range(2):  # the first run warms up
        ek[0].record()
        vsd.sample_score_paths(prob, params_kl, Xs, Ys, inp["d2t"], inp["valid_depth"], cfg.philox_seed,
                               cfg.philox_offset, out=out_kl, workspace=ws, tokens=tok)
        ek[1].record()
        vsd.weighted_loss_bwd(prob, params_kl, Xs, out_kl.lse_draft, tok[0], tok[1], out_kl.coef_a, out_kl.coef_b,
                              grad=grad, device_error=err, kl_idx=out_kl.kl_idx, kl_grad=out_kl.kl_grad)
        ek[2].record()
    torch.cuda.synchronize()
    kl_variant = {"kl_topk": 10, "kl_weight": 0.1, "sample_score_ms": ek[0].elapsed_time(ek[1]),
                  "bwd_ms": ek[1].elapsed_time(ek[2]), "ms_per_step": ek[0].elapsed_time(ek[2])}
    if int(err.item()) != 0 or int(out.device_error.item()) != 0 or int(out_kl.device_error.item()) != 0:
        raise RuntimeError("device error reported during the LM-head benchmark")
    del out_kl
    live = prob.R if inp["valid_depth"] is None else int((tok[0] >= 0).sum().item())
    R, H = prob.R, cfg.hidden
    # algorithmic flops: every row's draft and target logits once (forward);
    # the draft logits again and g W_d (backward)
    fwd_flop = 2.0 * R * H * (cfg.v_draft + cfg.v_target)
    bwd_flop = 4.0 * R * H * cfg.v_draft
    tf = lambda f, ms: f / (ms * 1e-3) / 1e12
    res = {
        "workload": f"{cfg.name}: B={cfg.B} T={cfg.T} N={cfg.N} L={cfg.L} hidden={H} V_target={cfg.v_target} "
                    f"V_draft={cfg.v_draft} bf16 hidden states and LM-head weights",
        "path_tokens_per_step": live, "ms_per_step": t_fwd + t_bwd, "wall_ms_per_step": wall * 1e3 / steps,
        "value": live / ((t_fwd + t_bwd) * 1e-3), "unit": "path-tokens/s",
        "kernels": {"sample_score": {"ms": t_fwd, "flop": fwd_flop, "TFLOP/s": tf(fwd_flop, t_fwd)},
                    "bwd": {"ms": t_bwd, "flop": bwd_flop, "TFLOP/s": tf(bwd_flop, t_bwd)},
                    "bwd_with_weight_grad": {"ms": t_bwd_w, "flop": bwd_flop * 1.5,
                                             "TFLOP/s": tf(bwd_flop * 1.5, t_bwd_w)}},
        "step_TFLOP/s": tf(fwd_flop + bwd_flop, t_fwd + t_bwd),
        "kl_variant": kl_variant,
        "roofline": {"bound": "mfma", "kernel": "k_lm_fwd (forward call: GEMM tiles + sampling epilogue)",
                     "achieved": tf(fwd_flop, t_fwd), "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                     "frac": tf(fwd_flop, t_fwd) / MFMA_BF16_PEAK_TFLOPS,
                     "traffic": measured_traffic(cfg.name, "lm_fwd")},
    }
    rec = profile_record("mfma", cfg.name, "lm_fwd")
    if rec is not None:  # SQ_VALU_MFMA_BUSY_CYCLES / (GRBM_GUI_ACTIVE per XCD x 1024 SIMDs), same sources
        res["roofline"]["mfma_counters"] = {"busy": rec["mfma_busy"], "clock_GHz": rec["clock_GHz"]}
    del inp, out, ws, grad
    torch.cuda.empty_cache()
    return res


PROFILE_FILES = [os.path.join(ROOT, "profiles", f) for f in ("c3_hbm_traffic.md", "lm_head_c5.md",
                                                               "c3_sample_score_valu.md")]
KERNEL_SOURCES = {"sample_score": ["k_sample.hip", "vsd_draw.hpp", "vsd_topk.hpp", "vsd_device.hpp", "vsd_kernels.hpp"],
                  "bwd": ["k_bwd.hip", "vsd_topk.hpp", "vsd_device.hpp", "vsd_kernels.hpp"],
                  "lm_fwd": ["k_lmhead.hip", "vsd_device.hpp", "vsd_kernels.hpp"]}


def source_hash(kernel):
    """Hash of the sources a kernel is built from (traffic figures go stale when it changes)."""
    import hashlib
    h = hashlib.sha256()
    for f in KERNEL_SOURCES[kernel]:
        with open(os.path.join(ROOT, "paper_2602_05774_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


def profile_record(tag, workload, kernel):
    """The machine-readable `tag:` record of a PMC summary in profiles/ for
    this workload and kernel, or None when there is none or the kernel's
    sources changed since the counters were taken."""
    for path in PROFILE_FILES:
        if not os.path.exists(path):
            continue
        for line in open(path):
            if line.startswith(tag + ":"):
                rec = json.loads(line[len(tag) + 1:])
                if rec.get("workload") == workload and rec.get("kernel") == kernel:
                    return rec if rec.get("source_hash") == source_hash(kernel) else None
    return None


def measured_traffic(workload, kernel):
    """HBM bytes per launch (FETCH_SIZE + WRITE_SIZE, calibrated) from the PMC
    summaries in profiles/, or None."""
    rec = profile_record("traffic", workload, kernel)
    return None if rec is None else rec.get("bytes_per_launch")


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--config", default="C3")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-workers", type=int, default=0)
    ap.add_argument("--no-lm-head", action="store_true", help="skip the fused LM-head measurement")
    ap.add_argument("--lm-steps", type=int, default=3, help="timed steps of the fused LM-head measurement")
    ap.add_argument("--no-ctx", action="store_true", help="skip the exact-context measurement")
    ap.add_argument("--no-configs", action="store_true", help="skip the C2 and C4 measurements")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="run one plain device copy of this size first (calibrates PMC byte counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU; --gpus {args.gpus} is not supported (positions shard "
              "independently across GPUs; run one process per GPU).", file=sys.stderr)
        sys.exit(2)

    from synth import CONFIGS
    cfg = CONFIGS[args.config]
    if cfg.kind == "fused":
        main_lm_head(args, cfg)
        return

    base = None
    if not args.no_cpu_baseline:
        workers = args.cpu_workers or default_workers()
        base = cpu_baseline(cfg, workers)
        print(f"[bench] cpu baseline: {base['value']:.1f} {base['unit']} on {base['cores']} cores", flush=True)

    import torch

    import paper_2602_05774_amd as vsd
    from synth import make_inputs

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    t0 = time.perf_counter()
    inp = make_inputs(cfg, dev)
    torch.cuda.synchronize()
    print(f"[bench] inputs {cfg.name} generated in {time.perf_counter() - t0:.1f} s", flush=True)
    prob = vsd.Problem(cfg.B, cfg.T, cfg.N, cfg.L, cfg.v_draft, cfg.v_target)
    params = vsd.Params(temp_draft=cfg.temp_draft, temp_target=cfg.temp_target)
    X, Y, d2t, depth = inp["X"], inp["Y"], inp["d2t"], inp["valid_depth"]
    out = vsd.alloc_score_outputs(prob, dev)
    ws = torch.empty(vsd.score_workspace_bytes(prob, X.dtype), dtype=torch.uint8, device=dev)
    grad = torch.empty_like(X)
    err = torch.zeros(1, dtype=torch.int32, device=dev)

    tok = [torch.empty(prob.R, dtype=torch.int32, device=dev) for _ in range(3)]
    if args.copy_calibration_mib:
        copy_calibration(args.copy_calibration_mib, dev)

    def step_fused(ev=None):
        """One EM step: one-pass sample + score, then the backward."""
        if ev:
            ev[0].record()
        vsd.sample_score_paths(prob, params, X, Y, d2t, depth, cfg.philox_seed, cfg.philox_offset, out=out,
                               workspace=ws, tokens=tok)
        if ev:
            ev[1].record()
        vsd.weighted_loss_bwd(prob, params, X, out.lse_draft, tok[0], tok[1], out.coef_a, out.coef_b, grad=grad,
                              device_error=err)
        if ev:
            ev[2].record()

    def step_three_calls(ev=None):
        """The same step through the three separate calls."""
        if ev:
            ev[0].record()
        s = vsd.sample_paths(prob, X, Y, d2t, depth, cfg.temp_draft, cfg.temp_target, cfg.philox_seed,
                             cfg.philox_offset, device_error=err)
        if ev:
            ev[1].record()
        vsd.score_paths(prob, params, X, Y, s.tok_draft, s.tok_target, s.tok_greedy, d2t, depth, out=out,
                        workspace=ws)
        if ev:
            ev[2].record()
        vsd.weighted_loss_bwd(prob, params, X, out.lse_draft, s.tok_draft, s.tok_target, out.coef_a, out.coef_b,
                              grad=grad, device_error=err)
        if ev:
            ev[3].record()

    def timed(fn, nev):
        for _ in range(args.warmup):
            fn()
        torch.cuda.synchronize()
        evs = [[torch.cuda.Event(enable_timing=True) for _ in range(nev)] for _ in range(args.steps)]
        t0 = time.perf_counter()
        for k in range(args.steps):
            fn(evs[k])
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        seg = [sum(e[j].elapsed_time(e[j + 1]) for e in evs) / args.steps for j in range(nev - 1)]
        total = sum(e[0].elapsed_time(e[nev - 1]) for e in evs) / args.steps
        return seg, total, wall

    params_kl = vsd.Params(temp_draft=cfg.temp_draft, temp_target=cfg.temp_target, kl_weight=0.1, kl_topk=10)
    out_kl = vsd.alloc_score_outputs(prob, dev, kl_topk=params_kl.kl_topk)

    def step_kl(ev=None):
        """The three-call step with the top-K renormalised KL term on."""
        if ev:
            ev[0].record()
        s = vsd.sample_paths(prob, X, Y, d2t, depth, cfg.temp_draft, cfg.temp_target, cfg.philox_seed,
                             cfg.philox_offset, device_error=err)
        if ev:
            ev[1].record()
        vsd.score_paths(prob, params_kl, X, Y, s.tok_draft, s.tok_target, s.tok_greedy, d2t, depth, out=out_kl,
                        workspace=ws)
        if ev:
            ev[2].record()
        vsd.weighted_loss_bwd(prob, params_kl, X, out_kl.lse_draft, s.tok_draft, s.tok_target, out_kl.coef_a,
                              out_kl.coef_b, grad=grad, device_error=err, kl_idx=out_kl.kl_idx,
                              kl_grad=out_kl.kl_grad)
        if ev:
            ev[3].record()

    tok_kl = [torch.empty(prob.R, dtype=torch.int32, device=dev) for _ in range(3)]

    def step_kl_fused(ev=None):
        """The one-pass step with the top-K renormalised KL term on."""
        if ev:
            ev[0].record()
        vsd.sample_score_paths(prob, params_kl, X, Y, d2t, depth, cfg.philox_seed, cfg.philox_offset, out=out_kl,
                               workspace=ws, tokens=tok_kl)
        if ev:
            ev[1].record()
        vsd.weighted_loss_bwd(prob, params_kl, X, out_kl.lse_draft, tok_kl[0], tok_kl[1], out_kl.coef_a,
                              out_kl.coef_b, grad=grad, device_error=err, kl_idx=out_kl.kl_idx,
                              kl_grad=out_kl.kl_grad)
        if ev:
            ev[2].record()

    (t_sample3, t_score3, t_bwd3), t_step3, _ = timed(step_three_calls, 4)
    (_, t_score_kl, t_bwd_kl), t_step_kl, _ = timed(step_kl, 4)
    (t_ss_kl, t_bwd_kl1), t_step_kl1, _ = timed(step_kl_fused, 3)
    (t_ss, t_bwd), t_step, wall = timed(step_fused, 3)
    if int(err.item()) != 0 or int(out.device_error.item()) != 0 or int(out_kl.device_error.item()) != 0:
        raise RuntimeError("device error reported during the benchmark")

    live = prob.R if depth is None else int((tok[0] >= 0).sum().item())
    nonzero = int(((out.coef_a != 0) | (out.coef_b != 0)).sum().item())
    es = X.element_size()
    # algorithmic bytes per launch: every live row's draft and target logits
    # once (sample + score), the backward's read of rows with a or b != 0 and
    # its write of every row
    ss_bytes = live * es * (cfg.v_draft + cfg.v_target)
    bwd_bytes = nonzero * es * cfg.v_draft + prob.R * es * cfg.v_draft
    gbs = lambda b, ms: b / (ms * 1e-3) / 1e9
    kernels = {
        "sample_score": {"ms": t_ss, "bytes": ss_bytes, "GB/s": gbs(ss_bytes, t_ss)},
        "bwd": {"ms": t_bwd, "bytes": bwd_bytes, "GB/s": gbs(bwd_bytes, t_bwd)},
    }
    three_calls = {"ms_per_step": t_step3, "sample_ms": t_sample3, "score_ms": t_score3, "bwd_ms": t_bwd3,
                   "score_GB/s": gbs(ss_bytes, t_score3),
                   "score_bwd_frac_of_hbm_peak": gbs(ss_bytes + bwd_bytes, t_score3 + t_bwd3) / HBM_PEAK_GBS}
    # The essential VALU lane operations of the one-pass sampler per live row
    # (a model, reported beside the byte roofline): 4 per logit for the two
    # log-sum-exps (unpack, fma, exp2, add), 40 per Philox4x32-10 call (10
    # rounds of two 32x32->64 products and two 3-way XORs; ceil(V_d/4) calls
    # per family, two families) and 14 per 8-key slice for the candidate bound.
    ss_ops = live * (4.0 * (cfg.v_draft + cfg.v_target) + 40.0 * 2 * ((cfg.v_draft + 3) // 4)
                     + 14.0 * 2 * ((cfg.v_draft + 7) // 8))
    kernels["sample_score"]["valu_model_lane_ops"] = ss_ops
    kernels["sample_score"]["valu_model_TOP/s"] = ss_ops / (t_ss * 1e-3) / 1e12
    kl_variant = {"kl_topk": params_kl.kl_topk, "kl_weight": params_kl.kl_weight,
                  "one_pass": {"ms_per_step": t_step_kl1, "path_tokens_per_s": live / (t_step_kl1 * 1e-3),
                               "sample_score_ms": t_ss_kl, "bwd_ms": t_bwd_kl1},
                  "three_calls": {"ms_per_step": t_step_kl, "score_ms": t_score_kl,
                                  "score_GB/s": gbs(ss_bytes, t_score_kl), "bwd_ms": t_bwd_kl,
                                  "bwd_GB/s": gbs(bwd_bytes, t_bwd_kl),
                                  "score_bwd_frac_of_hbm_peak": gbs(ss_bytes + bwd_bytes, t_score_kl + t_bwd_kl)
                                  / HBM_PEAK_GBS}}
    # Roofline of the step's dominant kernel against HBM: its algorithmic
    # bytes (every live row's draft and target logits read once for the
    # one-pass sampler; the backward's reads and writes) over its measured
    # time.  The one-pass sampler also runs close to the VALU issue limit: the
    # counter-based issue fraction (SQ_INSTS_VALU x 64 lanes over the time,
    # against 256 CUs x 4 SIMDs x 16 lanes x 2.4 GHz) comes from its profile
    # summary when that was taken on the current sources.
    dominant = "sample_score" if t_ss >= t_bwd else "bwd"
    k = kernels[dominant]
    roof = {"bound": "hbm", "kernel": "k_sample (one-pass sample + score, mapped, bf16)" if dominant == "sample_score"
            else "k_bwd", "achieved": k["GB/s"], "peak": HBM_PEAK_GBS, "unit": "GB/s",
            "frac": k["GB/s"] / HBM_PEAK_GBS, "traffic": measured_traffic(cfg.name, dominant),
            "bytes_per_launch": k["bytes"], "ms_per_launch": k["ms"]}
    if dominant == "sample_score":
        roof["valu_model"] = {"lane_ops_per_launch": ss_ops, "achieved_TOP/s": k["valu_model_TOP/s"],
                              "issue_peak_TOP/s": VALU_PEAK_TOPS, "frac": k["valu_model_TOP/s"] / VALU_PEAK_TOPS}
        rec = profile_record("valu", cfg.name, dominant)
        if rec is not None:
            lane_ops = rec["sq_insts_valu"] * 64.0
            roof["valu_counters"] = {"sq_insts_valu": rec["sq_insts_valu"],
                                     "lane_ops_per_s": lane_ops / (k["ms"] * 1e-3),
                                     "frac_of_issue_peak": lane_ops / (k["ms"] * 1e-3) / (VALU_PEAK_TOPS * 1e12)}
    line = {
        "metric": METRIC, "value": live / (t_step * 1e-3), "unit": "path-tokens/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": t_step, "wall_ms_per_step": wall * 1e3 / args.steps,
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": f"{cfg.name}: B={cfg.B} T={cfg.T} N={cfg.N} L={cfg.L} "
                               f"V_target={cfg.v_target} V_draft={cfg.v_draft} logits={cfg.dtype}",
                   "path_tokens_per_step": live, "parallelism": "single GPU"},
        "kernels": kernels, "three_calls": three_calls, "kl_variant": kl_variant, "roofline": roof,
        "cpu_baseline": base,
    }
    ref = hbm_reference(dev)
    ref["score_frac_of_read"] = three_calls["score_GB/s"] / ref["read_GB/s"]
    line["hbm_reference"] = ref
    if roof.get("traffic"):  # the dominant kernel's measured fetch rate against the box's streaming read
        t_dom = kernels[dominant]["ms"]
        roof["traffic_GB/s"] = roof["traffic"] / (t_dom * 1e-3) / 1e9
        roof["traffic_frac_of_measured_read"] = roof["traffic_GB/s"] / ref["read_GB/s"]
    line["verification"] = bench_verify(cfg, prob, params, inp, out, ws, timed, dev)
    if not args.no_ctx:
        line["exact_context"] = bench_ctx(cfg, prob, params, inp, ws, timed, live, dev)
    del inp, X, Y, out, out_kl, ws, grad
    torch.cuda.empty_cache()
    if not args.no_configs:
        line["configs"] = {name: bench_config(CONFIGS[name], args.steps, args.warmup, dev)
                           for name in ("C2", "C4") if name != cfg.name}
    if not args.no_lm_head:
        line["fused_lm_head"] = bench_lm_head(CONFIGS["C5"], args.lm_steps, 1, dev)
    print(json.dumps(line), flush=True)


def time_calls(fn, nev, steps, warmup):
    """warmup untimed calls, then `steps` timed ones; fn(ev) records nev
    events on the current stream.  Returns (mean ms between consecutive
    events, mean ms first to last)."""
    import torch
    for _ in range(warmup):
        fn(None)
    torch.cuda.synchronize()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(nev)] for _ in range(steps)]
    for k in range(steps):
        fn(evs[k])
    torch.cuda.synchronize()
    seg = [sum(e[j].elapsed_time(e[j + 1]) for e in evs) / steps for j in range(nev - 1)]
    return seg, sum(e[0].elapsed_time(e[nev - 1]) for e in evs) / steps


def bench_config(cfg, steps, warmup, dev):
    """The EM step on another workload: the one-pass step (sample + score in
    one call, then the backward) and the graded score + backward of the three
    calls, with their HBM fractions (algorithmic bytes: every live row's draft
    and target logits once for sample + score or score; the backward reads the
    rows with a or b != 0 and writes every row)."""
    import torch

    import paper_2602_05774_amd as vsd
    from synth import make_inputs
    t0 = time.perf_counter()
    inp = make_inputs(cfg, dev)
    torch.cuda.synchronize()
    print(f"[bench] inputs {cfg.name} generated in {time.perf_counter() - t0:.1f} s", flush=True)
    prob = vsd.Problem(cfg.B, cfg.T, cfg.N, cfg.L, cfg.v_draft, cfg.v_target)
    params = vsd.Params(temp_draft=cfg.temp_draft, temp_target=cfg.temp_target)
    X, Y, d2t, depth = inp["X"], inp["Y"], inp["d2t"], inp["valid_depth"]
    out = vsd.alloc_score_outputs(prob, dev)
    ws = torch.empty(vsd.score_workspace_bytes(prob, X.dtype), dtype=torch.uint8, device=dev)
    grad = torch.empty_like(X)
    err = torch.zeros(1, dtype=torch.int32, device=dev)
    tok = [torch.empty(prob.R, dtype=torch.int32, device=dev) for _ in range(3)]

    def one_pass(ev):
        if ev:
            ev[0].record()
        vsd.sample_score_paths(prob, params, X, Y, d2t, depth, cfg.philox_seed, cfg.philox_offset, out=out,
                               workspace=ws, tokens=tok)
        if ev:
            ev[1].record()
        vsd.weighted_loss_bwd(prob, params, X, out.lse_draft, tok[0], tok[1], out.coef_a, out.coef_b, grad=grad,
                              device_error=err)
        if ev:
            ev[2].record()

    def three_calls(ev):
        if ev:
            ev[0].record()
        vsd.sample_paths(prob, X, Y, d2t, depth, cfg.temp_draft, cfg.temp_target, cfg.philox_seed,
                         cfg.philox_offset, tokens=tok, device_error=err)
        if ev:
            ev[1].record()
        vsd.score_paths(prob, params, X, Y, tok[0], tok[1], tok[2], d2t, depth, out=out, workspace=ws)
        if ev:
            ev[2].record()
        vsd.weighted_loss_bwd(prob, params, X, out.lse_draft, tok[0], tok[1], out.coef_a, out.coef_b, grad=grad,
                              device_error=err)
        if ev:
            ev[3].record()

    (t_sample3, t_score3, t_bwd3), t_step3 = time_calls(three_calls, 4, steps, warmup)
    (t_ss, t_bwd), t_step = time_calls(one_pass, 3, steps, warmup)
    if int(err.item()) != 0 or int(out.device_error.item()) != 0:
        raise RuntimeError(f"device error reported during the {cfg.name} benchmark")
    live = prob.R if depth is None else int((tok[0] >= 0).sum().item())
    nonzero = int(((out.coef_a != 0) | (out.coef_b != 0)).sum().item())
    es = X.element_size()
    ss_bytes = live * es * (cfg.v_draft + cfg.v_target)
    bwd_bytes = nonzero * es * cfg.v_draft + prob.R * es * cfg.v_draft
    gbs = lambda b, ms: b / (ms * 1e-3) / 1e9
    res = {"workload": f"{cfg.name}: B={cfg.B} T={cfg.T} N={cfg.N} L={cfg.L} V_target={cfg.v_target} "
                       f"V_draft={cfg.v_draft} logits={cfg.dtype} T_q={cfg.temp_draft}"
                       + (" ragged depths" if cfg.ragged else ""),
           "path_tokens_per_step": live, "ms_per_step": t_step, "value": live / (t_step * 1e-3),
           "unit": "path-tokens/s",
           "one_pass": {"sample_score_ms": t_ss, "bwd_ms": t_bwd, "sample_score_GB/s": gbs(ss_bytes, t_ss),
                        "bwd_GB/s": gbs(bwd_bytes, t_bwd)},
           "three_calls": {"ms_per_step": t_step3, "sample_ms": t_sample3, "score_ms": t_score3, "bwd_ms": t_bwd3,
                           "score_bytes": ss_bytes, "bwd_bytes": bwd_bytes,
                           "score_GB/s": gbs(ss_bytes, t_score3), "bwd_GB/s": gbs(bwd_bytes, t_bwd3),
                           "score_bwd_frac_of_hbm_peak": gbs(ss_bytes + bwd_bytes, t_score3 + t_bwd3)
                           / HBM_PEAK_GBS}}
    del inp, X, Y, out, ws, grad
    torch.cuda.empty_cache()
    return res


def hbm_reference(dev, gib=4):
    """Measured HBM rates of plain library kernels on this machine, as reference
    points for the roofline fractions: a streaming read (the faster of two
    integer reductions over a buffer of `gib` GiB, which read at the box's
    practical rate) and a device copy of half that size (read + write)."""
    import torch

    n = (gib << 30) // 2
    buf = torch.ones(n, dtype=torch.bfloat16, device=dev)
    dst = torch.empty(n // 2, dtype=torch.bfloat16, device=dev)

    def median_ms(fn, reps=7):
        fn()
        torch.cuda.synchronize()
        ts = []
        for _ in range(reps):
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            fn()
            e1.record()
            torch.cuda.synchronize()
            ts.append(e0.elapsed_time(e1))
        return sorted(ts)[reps // 2]

    t_read = min(median_ms(lambda: buf.view(torch.int64).sum()),
                 median_ms(lambda: buf.view(torch.int32).view(-1, 1 << 15).amax(dim=1)))
    t_copy = median_ms(lambda: dst.copy_(buf[: n // 2]))
    res = {"read_GB/s": 2 * n / (t_read * 1e-3) / 1e9, "copy_GB/s": 2 * (2 * (n // 2)) / (t_copy * 1e-3) / 1e9,
           "read_bytes": 2 * n, "kernels": "torch int64 sum / int32 row amax (read), copy_ (read + write)"}
    del buf, dst
    torch.cuda.empty_cache()
    return res


def bench_verify(cfg, prob, params, inp, out, ws, timed, dev):
    """Decode-time verification of the step's draft paths (vsd_verify_paths
    on the scores `out` holds).  Bytes: each rejected path's row is read once
    (target logits es V_t, draft logits es V_d through the inverse map)."""
    import torch

    import paper_2602_05774_amd as vsd
    X, Y, d2t, depth = inp["X"], inp["Y"], inp["d2t"], inp["valid_depth"]
    err = torch.zeros(1, dtype=torch.int32, device=dev)
    res = {}

    def step(ev=None):
        if ev:
            ev[0].record()
        res["v"] = vsd.verify_paths(prob, params, X, Y, out, d2t, depth, cfg.philox_seed, cfg.philox_offset,
                                    workspace=ws, device_error=err)
        if ev:
            ev[1].record()

    (t_verify,), _, _ = timed(step, 2)
    if int(err.item()) != 0:
        raise RuntimeError("device error reported during the verification benchmark")
    acc = res["v"].accept_len
    d = torch.full_like(acc, cfg.L) if depth is None else depth.reshape(-1)
    rejected = int((acc < d).sum().item())
    es = X.element_size()
    nbytes = rejected * es * (cfg.v_draft + cfg.v_target)
    return {"ms": t_verify, "paths": acc.numel(), "rejected_paths": rejected, "bytes": nbytes,
            "GB/s": nbytes / (t_verify * 1e-3) / 1e9, "mean_accept_len": float(acc.double().mean().item()),
            "mean_expected_accept_len": float(out.exp_accept_len.double().mean().item())}


def bench_ctx(cfg, prob, params, inp, ws, timed, live, dev):
    """The step with exact context on the same workload: each family has its
    own rows (two more copies of X and Y, distinct buffers), the draws go
    depth by depth (L vsd_sample_step calls), then vsd_score_paths_ctx and
    vsd_weighted_loss_bwd_ctx.  Bytes: scoring reads every live row of all
    three families, es (V_d + V_t) each; the backward reads the rows along z~
    (z') whose a (b) is nonzero and writes both gradients in full."""
    import torch

    import paper_2602_05774_amd as vsd
    from synth import depth_view
    X, Y, d2t, depth = inp["X"], inp["Y"], inp["d2t"], inp["valid_depth"]
    need = 2 * (X.numel() + Y.numel()) * X.element_size() + 2 * X.numel() * X.element_size()
    free, _ = torch.cuda.mem_get_info(dev)
    if free < need + (4 << 30):
        return {"skipped": f"needs {need / 2**30:.1f} GiB more device memory, {free / 2**30:.1f} free"}
    Xs = [X, X.clone(), X.clone()]
    Ys = [Y, Y.clone(), Y.clone()]
    grads = (torch.empty_like(X), torch.empty_like(X))
    out = vsd.alloc_score_outputs(prob, dev, full=False)
    out = out._replace(lse_draft_corr=torch.empty(prob.R, dtype=torch.float32, device=dev))
    toks = [torch.full((prob.R,), -1, dtype=torch.int32, device=dev) for _ in range(3)]
    err = torch.zeros(1, dtype=torch.int32, device=dev)
    n = cfg.P * cfg.N

    def step(ev=None):
        if ev:
            ev[0].record()
        for i in range(cfg.L):
            vsd.sample_step(prob, i, depth_view(Xs[0], n, cfg.L, i), depth_view(Ys[1], n, cfg.L, i),
                            depth_view(Ys[2], n, cfg.L, i), d2t, depth, cfg.temp_draft, cfg.temp_target,
                            cfg.philox_seed, cfg.philox_offset, tokens=toks, device_error=err)
        if ev:
            ev[1].record()
        vsd.score_paths_ctx(prob, params, Xs, Ys, *toks, d2t, depth, out=out, workspace=ws)
        if ev:
            ev[2].record()
        vsd.weighted_loss_bwd_ctx(prob, params, Xs, out.lse_draft, out.lse_draft_corr, toks[0], toks[1], out.coef_a,
                                  out.coef_b, grads=grads, device_error=err)
        if ev:
            ev[3].record()

    (t_sample, t_score, t_bwd), t_step, _ = timed(step, 4)
    if int(err.item()) != 0 or int(out.device_error.item()) != 0:
        raise RuntimeError("device error reported during the exact-context benchmark")
    es = X.element_size()
    na = int((out.coef_a != 0).sum().item())
    nb = int((out.coef_b != 0).sum().item())
    score_bytes = 3 * live * es * (cfg.v_draft + cfg.v_target)
    bwd_bytes = (na + nb) * es * cfg.v_draft + 2 * prob.R * es * cfg.v_draft
    gbs = lambda b, ms: b / (ms * 1e-3) / 1e9
    res = {"ms_per_step": t_step, "path_tokens_per_s": live / (t_step * 1e-3), "sample_steps_ms": t_sample,
           "score_ms": t_score, "score_bytes": score_bytes, "score_GB/s": gbs(score_bytes, t_score),
           "bwd_ms": t_bwd, "bwd_bytes": bwd_bytes, "bwd_GB/s": gbs(bwd_bytes, t_bwd),
           "score_bwd_frac_of_hbm_peak": gbs(score_bytes + bwd_bytes, t_score + t_bwd) / HBM_PEAK_GBS}
    del Xs, Ys, grads
    torch.cuda.empty_cache()
    return res


def main_lm_head(args, cfg):
    """--config C5: the fused LM-head step as the line's own workload."""
    base = None
    if not args.no_cpu_baseline:
        workers = args.cpu_workers or default_workers()
        base = cpu_baseline_lm(cfg, workers)
        print(f"[bench] cpu baseline: {base['value']:.2f} {base['unit']} on {base['cores']} cores", flush=True)
    import torch
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    if args.copy_calibration_mib:
        copy_calibration(args.copy_calibration_mib, dev)
    r = bench_lm_head(cfg, args.steps, args.warmup, dev)
    line = {
        "metric": METRIC, "value": r["value"], "unit": "path-tokens/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": r["ms_per_step"], "wall_ms_per_step": r["wall_ms_per_step"],
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16", "data": "synthetic",
        "config": {"workload": r["workload"], "path_tokens_per_step": r["path_tokens_per_step"],
                   "parallelism": "single GPU"},
        "kernels": r["kernels"], "step_TFLOP/s": r["step_TFLOP/s"], "kl_variant": r["kl_variant"],
        "roofline": r["roofline"], "cpu_baseline": base,
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
