"""Benchmark of one Domino draft step on one MI355X.

A step is domino_draft_step + domino_build_tree + domino_verify_accept on
inputs already resident in HBM (synthetic weights and context of the
Qwen3-8B shape, bs 1, context 1024, block 16, branch 1 by default).  Prints one
JSON line.  The CPU-baseline leg times the fp64 CPU oracle on a bounded sample
(one or more whole steps) on this machine's host cores.
"""
from __future__ import annotations

import argparse
import json
import os
import statistics
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK = 8.0e12  # B/s, MI355X HBM3E

# HBM bytes per LM-head launch from rocprofv3 FETCH_SIZE / WRITE_SIZE (scaled by a 1 GiB copy),
# valid for the GEMM source with this sha1 (see profiles/lm_head_gemm_qwen3_8b_bs1.md)
LMHEAD_TRAFFIC = {"gemm_sha1": "d9fa868d45f2fb76ea5d40388e30935f5d80b17d", "bytes": 1259095722,
                  "config": "qwen3_8b"}


PROF_EVERY = 10  # timed steps per LM-head launch bracketed by events


def lmhead_traffic(cfg_name):
    import hashlib
    src = os.path.join(ROOT, "paper_2605_29707_amd", "csrc", "gemm.hip")
    try:
        h = hashlib.sha1(open(src, "rb").read()).hexdigest()
    except OSError:
        return None
    if h != LMHEAD_TRAFFIC["gemm_sha1"] or cfg_name != LMHEAD_TRAFFIC["config"]:
        return None  # kernel changed since the counters were taken
    return LMHEAD_TRAFFIC["bytes"]


def algorithmic_bytes(cfg) -> dict:
    """Bytes a step must move at least: every weight once, the context KV, the
    target-logit rows the acceptance walk reads, the gathered embedding rows."""
    d, dh, nq, nkv, F, V = cfg.hidden, cfg.head_dim, cfg.n_q_heads, cfg.n_kv_heads, cfg.ffn, cfg.vocab
    ds, r, bs, B = cfg.gru_hidden, cfg.rank, cfg.batch, cfg.block
    es = 2 if cfg.dtype == "bf16" else 4
    layer = d * nq * dh + 2 * d * nkv * dh + nq * dh * d + 3 * d * F
    head = 3 * ds * d + 3 * ds * ds + r * (d + ds) + V * r
    parts = {
        "backbone": es * cfg.n_layers * layer,
        "lm_head": es * V * d,
        "domino_head": es * head,
        "ctx_kv": bs * cfg.n_layers * cfg.ctx * nkv * dh * 2 * es,
        "target_rows": bs * (B + (1 if cfg.branch > 1 else 0)) * V * 2,
        "embed_rows": bs * (2 * B - 1) * d * es,
    }
    parts["total"] = sum(parts.values())
    return parts


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--sample-steps", type=int, default=100,
                    help="extra steps at temperature 1: sampled drafting + tree + speculative-sampling "
                         "verification (reported per step; 0 skips)")
    ap.add_argument("--append-rows", type=int, default=4,
                    help="extra pass whose steps first append this many target hidden states to the context "
                         "KV cache of every layer (about tau of the previous cycle; 0 skips)")
    ap.add_argument("--train-steps", type=int, default=50,
                    help="extra pass timing the teacher-forced training forward + curriculum loss (0: skip)")
    ap.add_argument("--cycle-steps", type=int, default=20,
                    help="extra pass timing the full speculative cycle with a 36-layer Qwen3-8B-shaped target: "
                         "draft step, tree, target verify forward, acceptance, cache commit (0: skip)")
    ap.add_argument("--config", default="qwen3_8b")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="CPU-baseline sample: whole oracle steps until this much time has passed (min 2)")
    ap.add_argument("--breakdown", action="store_true", help="extra pass timing every kernel class")
    ap.add_argument("--calibrate-copy", type=int, default=0, metavar="MIB",
                    help="also run one plain device copy of MIB MiB (a known-size kernel for counter scaling)")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print(f"bench.py runs on one GPU: this build has no multi-GPU path (asked for {args.gpus}).",
              file=sys.stderr)
        sys.exit(2)

    import gc

    import torch

    import synth

    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    cfg = synth.get_config(args.config)
    t0 = time.time()
    w = synth.make_weights(cfg, seed=args.seed)
    inp = synth.make_inputs(cfg, seed=args.seed)
    print(f"# inputs generated in {time.time() - t0:.1f}s", file=sys.stderr, flush=True)
    res = run_gpu(args, cfg, w, inp)
    # Every device tensor of the run is gone with run_gpu's frame; hand the
    # cached blocks back to HIP now, while every runtime and any profiling tool
    # loaded into the process are still up, instead of at interpreter teardown.
    gc.collect()
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    torch.cuda.synchronize()
    if not args.no_cpu_baseline:
        res["cpu_baseline"] = cpu_baseline(cfg, w, inp, lg_seed=args.seed * 16, seconds=args.cpu_seconds)
    print(json.dumps(res), flush=True)


def run_gpu(args, cfg, w, inp):
    """Every GPU pass of the benchmark; returns the result record (without the CPU baseline)."""
    import torch

    import synth
    from paper_2605_29707_amd import binding as bd

    dev = torch.device("cuda:0")
    bs, D, beta, V = cfg.batch, cfg.depth, cfg.branch, cfg.vocab
    dw = bd.to_device_weights(w, cfg, dev)
    model = bd.DominoModel(cfg, dw)
    kvdt = torch.bfloat16 if cfg.dtype == "bf16" else torch.float32
    T = lambda a, dt=torch.float32: torch.from_numpy(np.ascontiguousarray(a)).to(dev).to(dt)
    anchor, lens = T(inp["anchor"], torch.int32), T(inp["ctx_lens"], torch.int32)
    ck, cv = T(inp["ctx_k"], kvdt), T(inp["ctx_v"], kvdt)
    hid = T(inp["ctx_hidden"]) if inp["ctx_hidden"] is not None else None
    n_new = 0 if hid is None else hid.shape[1]
    max_ctx = inp["max_ctx"]
    ws = torch.empty(model.workspace_bytes(bs, max_ctx, n_new, beta), dtype=torch.uint8, device=dev)
    ids = torch.empty(bs, D, beta, dtype=torch.int32, device=dev)
    vals = torch.empty(bs, D, beta, dtype=torch.float32, device=dev)
    nn = 1 + D * beta
    tok, par, dep, pos = (torch.empty(bs, nn, dtype=torch.int32, device=dev) for _ in range(4))
    acc = torch.empty(bs, dtype=torch.int32, device=dev)
    nodes = torch.empty(bs, D, dtype=torch.int32, device=dev)
    out = torch.empty(bs, D + 1, dtype=torch.int32, device=dev)
    vws = torch.empty(bd.domino_verify_workspace_bytes(bs, nn, V), dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream()

    def draft():
        bd.domino_draft_step(model, anchor, lens, ck, cv, max_ctx, ids, vals, ws, branch=beta,
                             ctx_hidden_new=hid, n_new=n_new, stream=stream)
        bd.domino_build_tree(ids, anchor, lens, tok, par, dep, pos, stream=stream)

    # target logits planted on this step's own tree (the step is deterministic); a few seeded
    # variants are cycled so acceptance lengths vary from step to step
    draft()
    torch.cuda.synchronize()
    targets = []
    for k in range(4):
        lg = synth.make_target_logits(cfg, tok.cpu().numpy(), par.cpu().numpy(), seed=args.seed * 16 + k,
                                      dtype="bf16")
        targets.append(T(lg, torch.bfloat16))
    del lg
    acc_hist = torch.zeros(len(targets), bs, dtype=torch.int32, device=dev)
    counter = [0]

    def step():
        draft()
        k = counter[0] % len(targets)
        counter[0] += 1
        bd.domino_verify_accept(tok, par, targets[k], cfg.block, acc, nodes, out, vws, stream=stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    assert bd.domino_workspace_error(ws) == 0, "device error word set"

    # timed region: K steps between two events; the LM-head launch of every PROF_EVERY-th step is
    # bracketed by library events (an event pair costs a few us of queue time, so not every step)
    dom = "lmhead"
    bd.domino_profile_enable(model, [dom])
    bd.domino_profile_reset(model)
    t0, t1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0.record(stream)
    for i in range(args.steps):
        bd.domino_profile_enable(model, [dom] if i % PROF_EVERY == 0 else [])
        step()
    t1.record(stream)
    torch.cuda.synchronize()
    total_ms = t0.elapsed_time(t1)
    dom_ms, dom_n = bd.domino_profile_read(model, dom)
    bd.domino_profile_enable(model, [])
    ms_per_step = total_ms / args.steps
    # the per-step distribution, from a second pass with an event after every step
    nd = min(args.steps, 100)
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(nd + 1)]
    torch.cuda.synchronize()
    evs[0].record(stream)
    for i in range(nd):
        step()
        evs[i + 1].record(stream)
    torch.cuda.synchronize()
    per = [evs[i].elapsed_time(evs[i + 1]) for i in range(nd)]
    taus = []
    for k in range(len(targets)):  # tau of each target variant (outside the timed region)
        bd.domino_verify_accept(tok, par, targets[k], cfg.block, acc, nodes, out, vws, stream=stream)
        torch.cuda.synchronize()
        taus += (acc.cpu().numpy() + 1).tolist()
    tau = float(np.mean(taus))

    sampled = None
    if args.sample_steps > 0 and beta == 1:
        final = torch.empty(bs, D, V, dtype=torch.float32, device=dev)
        sws = torch.empty(bd.domino_verify_sample_workspace_bytes(bs, cfg.block, V), dtype=torch.uint8, device=dev)

        def step_sampled(i):
            bd.domino_draft_step_sampled(model, anchor, lens, ck, cv, max_ctx, ids, vals, final, ws, 1.0,
                                         seed=1000 + i, ctx_hidden_new=hid, n_new=n_new, stream=stream)
            bd.domino_build_tree(ids, anchor, lens, tok, par, dep, pos, stream=stream)
            bd.domino_verify_sample(tok, targets[i % len(targets)], final, 1.0, 1000 + i, acc, nodes, out, sws,
                                    stream=stream)

        for i in range(5):
            step_sampled(i)
        se = [torch.cuda.Event(enable_timing=True) for _ in range(args.sample_steps + 1)]
        stau = torch.zeros(args.sample_steps, bs, dtype=torch.int32, device=dev)
        torch.cuda.synchronize()
        se[0].record(stream)
        for i in range(args.sample_steps):
            step_sampled(i)
            se[i + 1].record(stream)
            stau[i].copy_(acc)
        torch.cuda.synchronize()
        assert bd.domino_workspace_error(ws) == 0 and bd.domino_workspace_error(sws) == 0
        sper = [se[i].elapsed_time(se[i + 1]) for i in range(args.sample_steps)]
        sampled = {"temperature": 1.0, "steps": args.sample_steps,
                   "ms_per_step": round(se[0].elapsed_time(se[-1]) / args.sample_steps, 4),
                   "us_per_step_median": round(statistics.median(sper) * 1e3, 1),
                   "mean_tau_synthetic": round(float(stau.float().mean().item()) + 1.0, 3)}
        del final, sws

    # the headline pass: K steps, each after a 512 MiB scratch fill that evicts the
    # on-chip caches (L2 and the MALL), then a 512 MiB read of another buffer that
    # pushes the fill's dirty lines back to HBM (neither is timed; without the read the
    # step's first kernels would share HBM with that write-back), each step between two events
    scratch = torch.empty(512 * (1 << 20) // 4, dtype=torch.float32, device=dev)
    clean = torch.ones(512 * (1 << 20) // 4, dtype=torch.float32, device=dev)
    sink = torch.empty((), dtype=torch.float32, device=dev)
    fe = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(args.steps)]
    torch.cuda.synchronize()
    for i in range(args.steps):
        scratch.fill_(float(i))  # a fill kernel, not a memset
        torch.sum(clean, dim=0, out=sink)
        fe[i][0].record(stream)
        step()
        fe[i][1].record(stream)
    torch.cuda.synchronize()
    assert bd.domino_workspace_error(ws) == 0, "device error word set"
    fper = [a.elapsed_time(b) for a, b in fe]
    del scratch, clean, sink
    torch.cuda.empty_cache()

    appended = None
    if args.append_rows > 0 and hid is None:
        na = args.append_rows
        ah = T(synth.make_append_hidden(cfg, na, seed=args.seed))
        aws = torch.empty(model.workspace_bytes(bs, max_ctx, na, beta), dtype=torch.uint8, device=dev)

        def step_append():
            bd.domino_draft_step(model, anchor, lens, ck, cv, max_ctx, ids, vals, aws, branch=beta,
                                 ctx_hidden_new=ah, n_new=na, stream=stream)
            bd.domino_build_tree(ids, anchor, lens, tok, par, dep, pos, stream=stream)
            bd.domino_verify_accept(tok, par, targets[0], cfg.block, acc, nodes, out, vws, stream=stream)

        for _ in range(5):
            step_append()
        ae = [torch.cuda.Event(enable_timing=True) for _ in range(51)]
        torch.cuda.synchronize()
        ae[0].record(stream)
        for i in range(50):
            step_append()
            ae[i + 1].record(stream)
        torch.cuda.synchronize()
        assert bd.domino_workspace_error(aws) == 0
        aper = [ae[i].elapsed_time(ae[i + 1]) for i in range(50)]
        appended = {"rows": na, "fused_target_layers": cfg.ctx_fuse_layers, "steps": 50,
                    "ms_per_step": round(ae[0].elapsed_time(ae[-1]) / 50, 4),
                    "us_per_step_median": round(statistics.median(aper) * 1e3, 1)}
        if cfg.ctx_fuse_layers > 0:
            # the fusion launches (K-split GEMM + partial sum) bracketed by library events
            bd.domino_profile_enable(model, ["ctxproj"])
            for _ in range(10):
                step_append()
            torch.cuda.synchronize()
            fms, fn = bd.domino_profile_read(model, "ctxproj")
            bd.domino_profile_enable(model, [])
            kf = cfg.ctx_fuse_layers * cfg.hidden
            esz = 2 if cfg.dtype == "bf16" else 4
            fbytes = cfg.hidden * kf * esz + bs * na * (kf + cfg.hidden) * 4  # ctx_fc once, rows in and out
            fus = fms * 1e3 / max(fn, 1)
            appended["fusion"] = {"us": round(fus, 2), "launches": fn, "algorithmic_bytes": fbytes,
                                  "achieved_GBps": round(fbytes / (fus * 1e-6) / 1e9, 1),
                                  "hbm_frac": round(fbytes / (fus * 1e-6) / 8e12, 4)}
        del aws

    trained = None
    if args.train_steps > 0:
        import synth as _s
        labels = T(_s.make_forced_tokens(cfg, seed=args.seed), torch.int32)
        tws = torch.empty(bd.domino_train_workspace_bytes(model, bs, max_ctx, n_new), dtype=torch.uint8,
                          device=dev)
        tloss = torch.empty(3, dtype=torch.float32, device=dev)

        def step_train():
            bd.domino_train_forward(model, anchor, lens, ck, cv, max_ctx, labels, 0.5, float(D), tloss, tws,
                                    ctx_hidden_new=hid, n_new=n_new, stream=stream)

        for _ in range(5):
            step_train()
        nt = args.train_steps
        te = [torch.cuda.Event(enable_timing=True) for _ in range(nt + 1)]
        bd.domino_profile_enable(model, ["trainloss", "headloop"])
        bd.domino_profile_reset(model)
        torch.cuda.synchronize()
        te[0].record(stream)
        for i in range(nt):
            step_train()
            te[i + 1].record(stream)
        torch.cuda.synchronize()
        assert bd.domino_workspace_error(tws) == 0
        lms, ln = bd.domino_profile_read(model, "trainloss")
        hms, hn = bd.domino_profile_read(model, "headloop")
        bd.domino_profile_enable(model, [])
        tper = [te[i].elapsed_time(te[i + 1]) for i in range(nt)]
        t_s = te[0].elapsed_time(te[-1]) / nt / 1e3
        tbytes = algorithmic_bytes(cfg)
        tb = tbytes["total"] - tbytes["target_rows"]
        trained = {"steps": nt, "lambda": 0.5, "gamma": float(D), "ms_per_pass": round(t_s * 1e3, 4),
                   "us_per_pass_median": round(statistics.median(tper) * 1e3, 1),
                   "positions_per_s": round(bs * D / t_s, 1),
                   "hbm_roofline_frac": round(tb / t_s / HBM_PEAK, 4), "algorithmic_bytes": tb,
                   "state_recurrence_us": round(hms * 1e3 / max(1, hn), 1),
                   "w2_ce_loss_us": round(lms * 1e3 / max(1, ln), 1),
                   "loss": [round(float(x), 5) for x in tloss.cpu().tolist()]}
        del tws

    cycle = None
    if args.cycle_steps > 0 and cfg.name == "qwen3_8b":
        cycle = speculative_cycle(args, cfg, bd, torch, dev, stream, model, anchor, lens, ck, cv, max_ctx, ids, vals,
                                  ws, hid, n_new, beta)

    breakdown = None
    if args.breakdown:
        classes = [c for c in bd.KERNEL_CLASSES]
        bd.domino_profile_enable(model, classes)
        bd.domino_profile_reset(model)
        for _ in range(20):
            step()
        torch.cuda.synchronize()
        breakdown = {}
        for c in classes:
            ms, n = bd.domino_profile_read(model, c)
            if n:
                breakdown[c] = round(ms * 1000.0 / 20, 2)
        bd.domino_profile_enable(model, [])

    ab = algorithmic_bytes(cfg)
    flush_ms = float(np.mean(fper))
    step_s = flush_ms / 1e3
    warm_s = ms_per_step / 1e3
    dom_launch_s = dom_ms / 1e3 / max(1, dom_n)
    # LM head + W1's H half (fused into the same launch): weights once + fp32 H rows
    es = 2 if cfg.dtype == "bf16" else 4
    dom_bytes = ab["lm_head"] + es * cfg.rank * cfg.hidden + bs * D * cfg.hidden * 4
    achieved = dom_bytes / dom_launch_s / 1e9

    res = {
        "metric": "draft steps/sec + us/step (k=16, Qwen3-8B-shape, bs=1); % HBM roofline",
        "value": round(1.0 / step_s, 2),
        "unit": "draft steps/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(flush_ms, 4),
        "timing": "each timed step after a 512 MiB cache-evicting fill and a 512 MiB read of another buffer "
                  "(neither timed), between two HIP events",
        "us_per_step_median": round(statistics.median(fper) * 1e3, 1),
        "us_per_step_p10_p90": [round(float(np.percentile(fper, 10)) * 1e3, 1),
                                round(float(np.percentile(fper, 90)) * 1e3, 1)],
        "hbm_roofline_frac_step": round(ab["total"] / step_s / HBM_PEAK, 4),
        "warm": {"value": round(1.0 / warm_s, 2), "unit": "draft steps/s", "steps": args.steps,
                 "ms_per_step": round(ms_per_step, 4),
                 "timing": "K back-to-back steps between two HIP events, caches warm",
                 "us_per_step_median": round(statistics.median(per) * 1e3, 1),
                 "us_per_step_p10_p90": [round(float(np.percentile(per, 10)) * 1e3, 1),
                                         round(float(np.percentile(per, 90)) * 1e3, 1)],
                 "hbm_roofline_frac_step": round(ab["total"] / warm_s / HBM_PEAK, 4)},
        "algorithmic_bytes_per_step": ab["total"],
        "drafted_tokens_per_s": round(bs * D / step_s, 1),
        "mean_tau_synthetic": round(tau, 3),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg.dtype,
        "data": "synthetic (seeded N(0,0.02) weights, N(0,1) context KV, Zipf(1.1) target logits)",
        "config": {"workload": f"{cfg.name}: draft step + tree + greedy acceptance",
                   "batch": bs, "ctx": cfg.ctx, "block": cfg.block, "branch": beta,
                   "hidden": cfg.hidden, "layers": cfg.n_layers, "vocab": V,
                   "storage": cfg.dtype},
        "roofline": {"kernel": "LM-head GEMM (gemm_stream_kernel<bf16_t, 1, 16, 8, 5>, W1 H-half fused)", "bound": "hbm",
                     "achieved": round(achieved, 1), "peak": HBM_PEAK / 1e9, "unit": "GB/s",
                     "frac": round(achieved * 1e9 / HBM_PEAK, 4), "traffic": lmhead_traffic(cfg.name),
                     "launch_us": round(dom_launch_s * 1e6, 2), "launches": dom_n,
                     "algorithmic_bytes_per_launch": dom_bytes,
                     "step": {"bound": "hbm", "achieved": round(ab["total"] / step_s / 1e9, 1),
                              "peak": HBM_PEAK / 1e9, "unit": "GB/s",
                              "frac": round(ab["total"] / step_s / HBM_PEAK, 4),
                              "algorithmic_bytes": ab["total"]}},
    }
    if sampled:
        res["sampling_t1"] = sampled
    if appended:
        res["with_context_append"] = appended
    if trained:
        res["training_forward"] = trained
    if cycle:
        res["speculative_cycle"] = cycle
    if breakdown:
        res["breakdown_us_per_step"] = breakdown

    if args.calibrate_copy:
        n = args.calibrate_copy * (1 << 20) // 4
        src = torch.ones(n, dtype=torch.float32, device=dev)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        res["calibration_copy_bytes"] = n * 4
        del src, dst

    torch.cuda.synchronize()
    model.close()
    return res


def target_bytes(tc) -> int:
    """Bytes a verify forward must move: every target weight once, the context
    KV of every layer, the embedding rows of the nodes."""
    d, dh, nq, nkv, F, V = tc.hidden, tc.head_dim, tc.n_q_heads, tc.n_kv_heads, tc.ffn, tc.vocab
    layer = d * nq * dh + 2 * d * nkv * dh + nq * dh * d + 3 * d * F
    return 2 * (tc.n_layers * layer + V * d) + tc.batch * tc.n_layers * tc.ctx * nkv * dh * 2 * 2 + 16 * d * 2


def speculative_cycle(args, cfg, bd, torch, dev, stream, model, anchor, lens, ck, cv, max_ctx, ids, vals, ws, hid,
                      n_new, beta):
    """Draft step + tree + target verify forward + greedy acceptance + cache
    commit, with a 36-layer Qwen3-8B-shaped target (random weights: only the
    timing means anything; the target shares the drafter's embedding and LM head)."""
    import synth
    tc = synth.get_config("qwen3_8b_target").with_(batch=cfg.batch, ctx=cfg.ctx, branch=beta)
    t0 = time.time()
    tw = synth.make_target_weights(tc, seed=args.seed)
    nn = tc.n_nodes
    tinp = synth.make_inputs(tc, seed=args.seed, max_ctx=tc.ctx + nn)
    tdw = bd.to_device_weights(tw, tc, dev)
    del tw
    target = bd.DominoModel(tc, tdw, target=True)
    T = lambda a, dt=torch.float32: torch.from_numpy(np.ascontiguousarray(a)).to(dev).to(dt)
    tck, tcv = T(tinp["ctx_k"], torch.bfloat16), T(tinp["ctx_v"], torch.bfloat16)
    tmax = tinp["max_ctx"]
    del tinp
    print(f"# target ready in {time.time() - t0:.1f}s", file=sys.stderr, flush=True)
    bs, D = cfg.batch, cfg.depth
    tok, par, dep, pos = (torch.empty(bs, nn, dtype=torch.int32, device=dev) for _ in range(4))
    mask = torch.empty(bs, nn, nn, dtype=torch.uint8, device=dev)
    tws = torch.empty(bd.domino_target_workspace_bytes(target, bs, nn, tmax), dtype=torch.uint8, device=dev)
    lg = torch.empty(bs, nn, cfg.vocab, dtype=torch.bfloat16, device=dev)
    acc = torch.empty(bs, dtype=torch.int32, device=dev)
    nodes = torch.empty(bs, D, dtype=torch.int32, device=dev)
    out = torch.empty(bs, D + 1, dtype=torch.int32, device=dev)
    vws = torch.empty(bd.domino_verify_workspace_bytes(bs, nn, cfg.vocab), dtype=torch.uint8, device=dev)
    new_lens = torch.empty(bs, dtype=torch.int32, device=dev)

    def one(ev=None):
        bd.domino_draft_step(model, anchor, lens, ck, cv, max_ctx, ids, vals, ws, branch=beta,
                             ctx_hidden_new=hid, n_new=n_new, stream=stream)
        bd.domino_build_tree(ids, anchor, lens, tok, par, dep, pos, ancestor_mask=mask, stream=stream)
        if ev:
            ev[0].record(stream)
        bd.domino_target_verify(target, tok, pos, mask, lens, tck, tcv, tmax, lg, tws, stream=stream)
        if ev:
            ev[1].record(stream)
        bd.domino_verify_accept(tok, par, lg, cfg.block, acc, nodes, out, vws, stream=stream)
        bd.domino_target_commit(target, nn, lens, acc, nodes, tck, tcv, tmax, new_lens, tws, stream=stream)

    for _ in range(3):
        one()
    n = args.cycle_steps
    ce = [torch.cuda.Event(enable_timing=True) for _ in range(n + 1)]
    ve = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(n)]
    taus = torch.zeros(n, bs, dtype=torch.int32, device=dev)
    torch.cuda.synchronize()
    ce[0].record(stream)
    for i in range(n):
        one(ve[i])
        ce[i + 1].record(stream)
        taus[i].copy_(acc)
    torch.cuda.synchronize()
    assert bd.domino_workspace_error(tws) == 0 and bd.domino_workspace_error(ws) == 0
    cyc = [ce[i].elapsed_time(ce[i + 1]) for i in range(n)]
    ver = [a.elapsed_time(b) for a, b in ve]
    tb = target_bytes(tc)
    v_s = statistics.median(ver) / 1e3
    tau = float(taus.float().mean().item()) + 1.0
    res = {"steps": n, "target": f"{tc.n_layers} layers, d {tc.hidden}, {tc.n_q_heads}q/{tc.n_kv_heads}kv, "
                                 f"FFN {tc.ffn}, V {tc.vocab}, bf16, {nn} nodes, ctx {tc.ctx}",
           "us_per_cycle_median": round(statistics.median(cyc) * 1e3, 1),
           "us_verify_forward_median": round(v_s * 1e6, 1),
           "verify_hbm_roofline_frac": round(tb / v_s / HBM_PEAK, 4), "verify_algorithmic_bytes": tb,
           "mean_tau_random_target": round(tau, 3),
           "tokens_per_s": round(bs * tau / (statistics.median(cyc) / 1e3), 1)}
    target.close()
    del target, tdw, tck, tcv
    torch.cuda.empty_cache()
    return res


def cpu_baseline(cfg, w, inp, lg_seed, seconds):
    """The fp64 oracle, as it stands, timed on whole steps of the same workload."""
    import oracle
    import synth
    from threadpoolctl import threadpool_info

    w64 = oracle.as_f64_weights(w)
    pools = threadpool_info()
    cores = max([i.get("num_threads", 1) for i in pools] + [1])
    blas = [f"{i.get('internal_api')} {i.get('version')} ({i.get('threading_layer', '?')} threads: "
            f"{i.get('num_threads')})" for i in pools if i.get("user_api") == "blas"]
    model = "unknown"
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                model = line.split(":", 1)[1].strip()
                break
    except OSError:
        pass
    beta = cfg.branch
    times = []
    while len(times) < 2 or sum(times) < seconds:
        t0 = time.time()
        r = oracle.draft_step(cfg, w64, inp["anchor"], inp["ctx_lens"], inp["ctx_k"], inp["ctx_v"], beta,
                              ctx_hidden=inp["ctx_hidden"])
        tree = oracle.build_tree(r["topk_ids"], inp["anchor"], inp["ctx_lens"])
        t1 = time.time()
        lg = synth.make_target_logits(cfg, tree["node_token"], tree["node_parent"], seed=lg_seed, dtype="bf16")
        t2 = time.time()
        oracle.verify_accept(tree["node_token"], tree["node_parent"], lg, cfg.block)
        t3 = time.time()
        times.append((t1 - t0) + (t3 - t2))
    med = statistics.median(times)
    return {"value": round(1.0 / med, 4), "unit": "draft steps/s", "cores": cores, "kind": "oracle",
            "nproc": os.cpu_count(), "affinity_cpus": len(os.sched_getaffinity(0)), "cpu_model": model,
            "blas": blas,
            "sample": f"{len(times)} whole steps of the same workload ({sum(times):.1f} s of fp64 numpy "
                      f"oracle; median {med:.2f} s/step; weight conversion and target-logit generation "
                      f"excluded)"}


if __name__ == "__main__":
    main()
