"""Throughput of one batch super-tree verification step on one MI355X.

A step is the whole hot path over one batch: echo_gate -> echo_build_tree_mask
-> echo_tree_verify_attn -> echo_accept, on inputs already resident in HBM.
The default workload is the Qwen3-235B-A22B-shaped layer at batch 128 (tree
8x10, budget 256, 64 q / 4 kv heads, head_dim 128, prefixes 1024-8192).

Prints one JSON line with the metric (verified tree nodes per second), the
roofline of the main attention kernel (timed with HIP events on its stream)
and the CPU oracle timed on a bounded sample of the same workload.
"""
import argparse
import hashlib
import json
import os
import platform
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0
PEAK_BF16_TFLOPS = 2500.0
METRIC = "verified tree nodes/sec (gate+verify-attn+accept), % HBM / MFMA peak"


# Checkpoint tables for the gate policies other than plain top-B.  ln tau at
# depth d is a + b (d - 1), (a, b) placed near the median per-request layer
# maximum of each synthetic workload, so that about half of the requests stop
# at each checkpoint.
TAU_LINE = {"tiny": (-1.1, -0.55), "l8b": (-3.1, -2.5), "l70b": (-2.9, -2.6),
            "q235b": (-3.0, -2.65), "long": (-2.1, -1.6)}


def gate_checkpoints(policy, cfg_name, depth):
    """(depth, ln tau) pairs of a gate policy: 'sparse' = checkpoints at depths
    1, 3, 5 (the paper's sweet-spot form), 'dense' = every drafted depth,
    'fixed' = every drafted depth at one threshold; 'topb' = none."""
    if policy == "topb":
        return None
    a, b = TAU_LINE[cfg_name]
    lt = lambda d: a + b * (d - 1)
    if policy == "sparse":
        return [(d, lt(d)) for d in (1, 3, 5) if d <= depth]
    if policy == "dense":
        return [(d, lt(d)) for d in range(1, depth + 1)]
    if policy == "fixed":
        return [(d, lt(3)) for d in range(1, depth + 1)]
    raise ValueError(policy)


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def attn_algorithmic(batch, res, cfg):
    """Algorithmic HBM bytes and FLOPs of one attention call: the prefix K and V
    once (bf16), plus per verify slot its q, new k/v, fp32 output and LSE; FLOPs
    are 4 * D * Hq per visible key of every slot (QK^T and PV)."""
    import numpy as np
    qo = res["q_offsets"]
    P = batch["prefix_len"].astype(np.int64)
    n = np.diff(qo).astype(np.int64)
    nq = int(qo[-1])
    D, hq, hkv = cfg.head_dim, cfg.hq, cfg.hkv
    kv_bytes = 4 * hkv * D * int(P.sum())                 # prefix K + V, bf16
    row_bytes = nq * (2 * hq * D + 4 * hkv * D + 4 * hq * D + 4 * hq)  # q, k/v_new, out, lse
    # visible keys per slot: prefix + ancestors-or-self (popcount of its mask row)
    mask = res["tree_mask"][:nq]
    anc = np.unpackbits(mask.view(np.uint8), axis=1).sum(axis=1).astype(np.int64)
    slot_req = np.repeat(np.arange(cfg.R), n)
    keys = P[slot_req] + anc
    flops = 4 * D * hq * int(keys.sum())
    return kv_bytes + row_bytes, flops


def attn_source_hash():
    """sha256 of what the attention kernel is built from: its source, the header with
    its workspace layout and plan, and the build script (which holds its compiler
    flags)."""
    h = hashlib.sha256()
    for rel in (("paper_2604_09603_amd", "csrc", "attn.hip"),
                ("paper_2604_09603_amd", "csrc", "attn_device.h"),
                ("paper_2604_09603_amd", "build.py")):
        with open(os.path.join(ROOT, *rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


PMC_SUMMARY = os.path.join(ROOT, "profiles", "attn_main_q235b_pmc.json")


def traffic_from_profile(attn_src_hash, workload_key, path=PMC_SUMMARY):
    """HBM bytes per attention-kernel launch from the committed rocprofv3 PMC summary.

    None unless the counters were taken on this workload (config, seed, gate policy, KV
    layout, serving step) with the current attention source and build flags.
    """
    if not os.path.exists(path):
        return None
    with open(path) as f:
        d = json.load(f)
    if d.get("attn_src_sha256") != attn_src_hash or d.get("workload_key") != workload_key:
        return None
    return d.get("hbm_bytes_per_launch")


# MI355X shape used to normalise the counters: 8 XCDs of 32 CUs, 4 SIMDs per CU,
# 4 shader engines per XCD, shader clock 2.4 GHz.
N_XCD, N_SIMD, N_SE, CLOCK_HZ = 8, 1024, 32, 2.4e9


def _pmc_medians(d, kernel="attn_main_kernel"):
    """Median per dispatch of every counter of `kernel` in a rocprofv3 --pmc output dir."""
    import csv
    import glob
    import statistics
    vals = {}
    for f in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
        with open(f) as fh:
            for r in csv.DictReader(fh):
                if kernel in r["Kernel_Name"]:
                    vals.setdefault(r["Counter_Name"], []).append(float(r["Counter_Value"]))
    return {k: statistics.median(v) for k, v in vals.items()}, {k: len(v) for k, v in vals.items()}


def pmc_summary(args):
    """Counters of the attention kernel, normalised, written to <pmc_out>.json and .md.

    Normalisation: GRBM_GUI_ACTIVE is summed over the 8 XCDs (cycles of one XCD =
    GRBM_GUI_ACTIVE / 8); SQ_VALU_MFMA_BUSY_CYCLES sums the busy cycles of the matrix
    units of all 1024 SIMDs (16 per v_mfma_f32_16x16x32_bf16), so the MFMA busy
    fraction is SQ_VALU_MFMA_BUSY_CYCLES / (GRBM_GUI_ACTIVE / 8 * 1024); SQ_BUSY_CYCLES
    sums the 32 shader engines; SQ_WAVE_CYCLES and the SQ_WAIT_* counters count in the
    same (quad-cycle) unit per wave, so their ratio is the fraction of a wave's life
    spent waiting; instruction counts are per dispatch and divided by SQ_WAVES;
    SQ_INSTS_VALU_MFMA_MOPS_BF16 counts 512-FLOP units; FETCH_SIZE and WRITE_SIZE (KiB)
    are scaled by what they read for a plain device copy of known size."""
    counters, samples = {}, {}
    for d in args.pmc_summary:
        m, n = _pmc_medians(d)
        counters.update(m)
        samples.update(n)
    out = {"kernel": "attn_main_kernel",
           "workload_key": {"config": args.config, "seed": args.seed, "gate_policy": args.gate_policy,
                            "page_size": args.page_size, "serve": bool(args.serve)},
           "attn_src_sha256": attn_source_hash(), "counters_median_per_dispatch": counters,
           "dispatches_per_counter": samples, "commands": args.pmc_commands}
    c = counters.get
    der = {}
    if c("GRBM_GUI_ACTIVE"):
        cyc = c("GRBM_GUI_ACTIVE") / N_XCD
        der["kernel_cycles_per_xcd"] = cyc
        der["kernel_us_at_2400mhz"] = cyc / CLOCK_HZ * 1e6
        if c("SQ_VALU_MFMA_BUSY_CYCLES") is not None:
            der["mfma_busy_frac"] = c("SQ_VALU_MFMA_BUSY_CYCLES") / (cyc * N_SIMD)
        if c("SQ_BUSY_CYCLES") is not None:
            der["sq_busy_frac"] = c("SQ_BUSY_CYCLES") / (cyc * N_SE)
        if c("SQ_INSTS_VALU_MFMA_MOPS_BF16") is not None:
            fl = c("SQ_INSTS_VALU_MFMA_MOPS_BF16") * 512.0
            der["mfma_flop_per_dispatch"] = fl
            der["mfma_tflops"] = fl / (cyc / CLOCK_HZ) / 1e12
    if c("SQ_WAVE_CYCLES"):
        for k in ("SQ_WAIT_INST_ANY", "SQ_WAIT_ANY", "SQ_ACTIVE_INST_VALU"):
            if c(k) is not None:
                der[k.lower() + "_per_wave_cycle"] = c(k) / c("SQ_WAVE_CYCLES")
    if c("SQ_WAVES"):
        for k in ("SQ_INSTS_VALU", "SQ_INSTS_MFMA", "SQ_INSTS_SALU", "SQ_INSTS_LDS", "SQ_INSTS_VMEM",
                  "SQ_INSTS_BRANCH", "SQ_INSTS_SMEM"):
            if c(k) is not None:
                der[k.lower() + "_per_wave"] = c(k) / c("SQ_WAVES")
    if c("SQ_INSTS_LDS"):
        if c("SQ_LDS_BANK_CONFLICT") is not None:
            der["lds_bank_conflict_cycles_per_lds_inst"] = c("SQ_LDS_BANK_CONFLICT") / c("SQ_INSTS_LDS")
    if args.pmc_copy and c("FETCH_SIZE") is not None and c("WRITE_SIZE") is not None:
        cf, _ = _pmc_medians(args.pmc_copy[0], kernel="copyBuffer")
        cw, _ = _pmc_medians(args.pmc_copy[1], kernel="copyBuffer")
        fs = args.pmc_copy_bytes / 1024.0 / cf["FETCH_SIZE"]
        ws = args.pmc_copy_bytes / 1024.0 / cw["WRITE_SIZE"]
        der["copy_fetch_kib"] = cf["FETCH_SIZE"]
        der["copy_write_kib"] = cw["WRITE_SIZE"]
        der["fetch_scale"] = fs
        der["write_scale"] = ws
        out["hbm_bytes_per_launch"] = (c("FETCH_SIZE") * fs + c("WRITE_SIZE") * ws) * 1024.0
    out["derived"] = der
    with open(args.pmc_out + ".json", "w") as f:
        json.dump(out, f, indent=1)
    from synth.configs import DESCRIPTION
    lines = [f"# rocprofv3 counters of attn_main_kernel, {DESCRIPTION.get(args.config, args.config)}, "
             f"seed {args.seed}", "", "Passes (each its own run, from the repository root as $REPO):",
             "", "```"] + list(args.pmc_commands) + ["```", "",
             "| counter | median per dispatch |", "|---|---|"]
    lines += [f"| {k} | {v:.0f} |" for k, v in sorted(counters.items())]
    lines += ["", "| derived | value |", "|---|---|"]
    lines += [f"| {k} | {v:.4g} |" for k, v in der.items()]
    if "hbm_bytes_per_launch" in out:
        lines += [f"| hbm_bytes_per_launch | {out['hbm_bytes_per_launch'] / 1e9:.4f} GB |"]
    lines += ["", "Normalisation: " + " ".join(pmc_summary.__doc__.split("Normalisation: ")[1].split()),
              "", f"sha256 of attn.hip + attn_device.h + build.py at measurement: `{out['attn_src_sha256']}`", ""]
    with open(args.pmc_out + ".md", "w") as f:
        f.write("\n".join(lines))
    log(f"wrote {args.pmc_out}.json and .md")


def cpu_model():
    """The host CPU's model name (from /proc/cpuinfo) and the cores this process may use."""
    name = platform.processor() or "unknown"
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    name = line.split(":", 1)[1].strip()
                    break
    except OSError:
        pass
    return name, len(os.sched_getaffinity(0))


def _oracle_front(batch, cfg, checkpoints, elastic):
    """The oracle's gate, mask and accept on the whole batch (single-threaded)."""
    import numpy as np

    import oracle
    import synth
    if elastic is not None:
        g = oracle.elastic_schedule(batch["cand_offsets"], batch["parent"], batch["logq"],
                                    cfg.budget, [d for d, _ in checkpoints],
                                    np.array([t for _, t in checkpoints], np.float32),
                                    elastic[0], elastic[1])
    elif checkpoints is None:
        g = oracle.gate(batch["cand_offsets"], batch["parent"], batch["logq"], cfg.budget)
    else:
        g = oracle.gate_sparse(batch["cand_offsets"], batch["parent"], batch["logq"],
                               cfg.budget, [d for d, _ in checkpoints],
                               np.array([t for _, t in checkpoints], np.float32))
    m = oracle.build_tree_mask(batch["cand_offsets"], batch["parent"], batch["token"],
                               g["selected"], batch["root_token"], batch["prefix_len"],
                               cfg.budget, cfg.mask_words)
    tgt = synth.target_for_slots(batch, m["q_offsets"], m["slot_cand"])
    oracle.accept(m["q_offsets"], m["slot_parent"], m["slot_token"], tgt, 16)
    return m


def _oracle_attn_requests(batch, cfg, m, reqs, budget_s):
    """Float64 oracle attention request by request until budget_s seconds are
    spent; returns (prefix-key work done, seconds, requests done)."""
    import numpy as np

    import oracle
    qo = m["q_offsets"]
    P = batch["prefix_len"].astype(np.int64)
    n = np.diff(qo)
    work, spent, done = 0.0, 0.0, 0
    for r in reqs:
        t1 = time.perf_counter()
        oracle.tree_verify_attn(batch["q"], batch["k_new"], batch["v_new"], batch["k_cache"],
                                batch["v_cache"], batch["kv_offsets"], qo, m["tree_mask"],
                                cfg.hq, cfg.hkv, batch["sm_scale"],
                                rows=range(int(qo[r]), int(qo[r + 1])))
        spent += time.perf_counter() - t1
        work += float(P[r] * n[r])
        done += 1
        if spent >= budget_s:
            break
    return work, spent, done


# inputs of the forked oracle workers (set before the pool forks, read-only there)
_WORKER_STATE = {}


def _oracle_worker(reqs):
    """One process of the all-cores leg: its share of the requests, again and again
    until the time budget is spent; returns (work, seconds, passes, start, end)
    with start and end on the host's monotonic clock."""
    from threadpoolctl import threadpool_limits
    st = _WORKER_STATE
    work, spent, done = 0.0, 0.0, 0
    start = time.perf_counter()
    with threadpool_limits(limits=1):
        while reqs and spent < st["budget_s"]:
            w, t, n = _oracle_attn_requests(st["batch"], st["cfg"], st["m"], reqs,
                                            st["budget_s"] - spent)
            work, spent, done = work + w, spent + t, done + n
    return work, spent, done, start, time.perf_counter()


def cpu_baseline(batch, cfg, checkpoints=None, elastic=None, budget_s=12.0, par_budget_s=8.0):
    """The oracle as written, timed on the host on a bounded sample of the workload.

    One-core leg: gate + mask + accept on the whole batch, then float64 attention
    request by request for about budget_s seconds; the attention time is scaled
    by prefix-key work to the whole step.  All-cores leg: the same attention
    spread over one process per usable core (at most 16), each over its share of
    the requests for about par_budget_s seconds; the aggregate rate is scaled the
    same way.  Runs before the GPU is touched, so that the workers can fork.
    """
    import multiprocessing

    import numpy as np
    from threadpoolctl import threadpool_limits

    model, usable = cpu_model()
    with threadpool_limits(limits=1):
        t0 = time.perf_counter()
        m = _oracle_front(batch, cfg, checkpoints, elastic)
        t_front = time.perf_counter() - t0
        qo = m["q_offsets"]
        P = batch["prefix_len"].astype(np.int64)
        work_all = float((P * np.diff(qo)).sum())
        order = np.random.default_rng(0).permutation(cfg.R)
        w1, t1, n1 = _oracle_attn_requests(batch, cfg, m, order, max(budget_s - t_front, 0.5))
    nq = int(qo[-1])
    est1 = t_front + t1 * work_all / max(w1, 1.0)
    procs = max(1, min(16, usable, cfg.R))
    _WORKER_STATE.update(batch=batch, cfg=cfg, m=m, budget_s=par_budget_s)
    shares = [order[i::procs].tolist() for i in range(procs)]
    ctx = multiprocessing.get_context("fork")
    with ctx.Pool(procs) as pool:
        parts = pool.map(_oracle_worker, shares, chunksize=1)
    # from the first worker's start to the last one's end (process start-up excluded)
    wall = max(p[4] for p in parts) - min(p[3] for p in parts)
    _WORKER_STATE.clear()
    wp = sum(p[0] for p in parts)
    np_done = sum(p[2] for p in parts)
    est_p = t_front + wall * work_all / max(wp, 1.0)
    return {
        "value": nq / est1, "unit": "verified tree nodes/sec", "cores": 1, "kind": "oracle",
        "cpu_model": model, "usable_cores": usable,
        "all_cores": {"value": nq / est_p, "unit": "verified tree nodes/sec", "cores": procs,
                      "processes": procs},
        "sample": (f"one core: oracle gate+mask+accept on the full batch ({t_front:.2f} s) and "
                   f"float64 attention for {n1} of {cfg.R} requests ({t1:.2f} s, "
                   f"{100.0 * w1 / work_all:.1f}% of the prefix-key work), attention scaled by "
                   f"prefix-key work to the whole step ({est1:.1f} s); all cores: the same "
                   f"attention over {procs} forked processes, each cycling through its share "
                   f"of the requests: {np_done} request passes, {100.0 * wp / work_all:.1f}% of "
                   f"the step's prefix-key work, in {wall:.2f} s wall; scaled the same way "
                   f"({est_p:.2f} s)"),
    }


def _pct(xs, q):
    import numpy as np
    return float(np.percentile(np.asarray(xs, np.float64), q))


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--config", default="q235b")
    ap.add_argument("--seed", type=int, default=3)
    ap.add_argument("--flush-mb", type=int, default=512,
                    help="MiB of device memory written, and as many read, between timed steps "
                         "(excluded from the timing) so that every step starts with the caches "
                         "holding other, clean data; 0 = back-to-back steps only")
    ap.add_argument("--protocol-steps", type=int, default=200,
                    help="cold steps behind the reported percentiles (at least --steps)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--gate-policy", default="topb",
                    choices=["topb", "sparse", "dense", "fixed", "elastic"],
                    help="gate stage: global top-B (default), checkpoint gating before it, or "
                         "Alg. 1's elastic scheduler (checkpoints at depths 1, 3, 5, W_topk = 2, "
                         "W_max = the drafted branching)")
    ap.add_argument("--page-size", type=int, default=0,
                    help="read the KV prefixes from a paged cache with pages of this many rows "
                         "(echo_tree_verify_attn_paged); 0 = contiguous")
    ap.add_argument("--serve", action="store_true",
                    help="the serving step: paged cache (64-row pages unless --page-size), "
                         "acceptance from bf16 target logits (echo_accept_logits) and the KV "
                         "commit of the accepted path (echo_commit_kv)")
    ap.add_argument("--separate-calls", action="store_true",
                    help="time the step as the four calls (gate, mask, attention, accept) "
                         "instead of the one echo_verify_step call")
    ap.add_argument("--graph", action="store_true",
                    help="capture one step in a HIP graph and time graph replays")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="BYTES",
                    help="only run a plain device-to-device copy of BYTES, five times (the "
                         "reference kernel that scales the HBM byte counters)")
    ap.add_argument("--pmc-summary", nargs="+", metavar="DIR",
                    help="only summarise rocprofv3 --pmc output directories of the attention "
                         "kernel (the counter passes of --config/--seed, then the FETCH_SIZE and "
                         "WRITE_SIZE passes of --copy-calibration) into --pmc-out .json/.md")
    ap.add_argument("--pmc-copy", nargs=2, metavar=("FETCH_DIR", "WRITE_DIR"),
                    help="with --pmc-summary: the copy-calibration passes")
    ap.add_argument("--pmc-copy-bytes", type=int, default=1 << 30)
    ap.add_argument("--pmc-out", default=None, help="path prefix of the summary files")
    ap.add_argument("--pmc-commands", nargs="*", default=[],
                    help="the commands that produced the passes (recorded in the summary)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (asked for --gpus {args.gpus}): the verification "
              "step runs on a single MI355X and there is no multi-GPU path.", file=sys.stderr)
        sys.exit(2)

    import numpy as np

    if args.pmc_summary:
        pmc_summary(args)
        return

    if args.copy_calibration > 0:
        import torch
        src = torch.empty(args.copy_calibration, dtype=torch.uint8, device="cuda:0")
        dst = torch.empty_like(src)
        src.fill_(1)
        torch.cuda.synchronize()
        for _ in range(5):
            dst.copy_(src)
        torch.cuda.synchronize()
        log(f"copied {args.copy_calibration} bytes five times")
        return

    import synth

    cfg = synth.CONFIGS[args.config]
    log(f"generating {args.config} seed={args.seed}")
    t0 = time.time()
    batch = synth.make_batch(args.config, args.seed)
    log(f"generated in {time.time() - t0:.1f} s")
    elastic = None
    if args.gate_policy == "elastic":
        checkpoints = gate_checkpoints("sparse", args.config, cfg.depth)
        elastic = (2, cfg.branch)
    else:
        checkpoints = gate_checkpoints(args.gate_policy, args.config, cfg.depth)
    cpu = None
    if not args.no_cpu_baseline:
        # before the GPU is touched: the all-cores leg forks worker processes
        log("timing the CPU oracle on a bounded sample")
        cpu = cpu_baseline(batch, cfg, checkpoints, elastic)

    import torch

    import paper_2604_09603_amd as pkg
    from paper_2604_09603_amd.step import VerifyStep

    log("uploading")
    page_size = args.page_size or (64 if args.serve else 0)
    st = VerifyStep(batch, device="cuda:0", checkpoints=checkpoints, elastic=elastic,
                    page_size=page_size or None, serve=args.serve)
    # the target model's argmax per slot is a stand-in input: gather it once for this batch
    st.gate()
    st.mask()
    torch.cuda.synchronize()
    res0 = st.fetch()
    tgt = synth.target_for_slots(batch, res0["q_offsets"], res0["slot_cand"])
    st.set_target(tgt)
    if args.serve:
        # synthetic target logits whose argmax is the stand-in target of each slot
        gen = torch.Generator(device="cuda:0")
        gen.manual_seed(args.seed)
        logits = torch.randn((st.cap, cfg.vocab), generator=gen, device="cuda:0")
        rows = torch.arange(len(tgt), device="cuda:0")
        logits[rows, torch.from_numpy(tgt.astype(np.int64)).to("cuda:0")] = 8.0
        st.set_logits(logits.to(torch.bfloat16))
        del logits
    flush = flush_src = None
    sink = torch.zeros(1, dtype=torch.int32, device="cuda:0")
    if args.flush_mb > 0:
        # the flush writes one buffer and then streams another one in with the
        # read probe's allocating copies, so that the caches hold clean lines of
        # unrelated data.  A write alone leaves up to a MALL's worth of dirty lines
        # whose write-back then lands inside the next step: head-strided copies
        # after a 512 MiB write read 4.6 TB/s instead of 6.0, which a serving loop
        # (weight reads and small activation writes between two attention calls of
        # a layer) does not see.  That case is reported separately.
        flush = torch.empty(args.flush_mb << 20, dtype=torch.uint8, device="cuda:0")
        flush_src = torch.ones(args.flush_mb << 20, dtype=torch.uint8, device="cuda:0")
        half = flush_src.view(2, -1)
        flush_rows = half.shape[1] // (4 * 256)
    torch.cuda.synchronize()

    # the step: one echo_verify_step call where it covers the configuration (top-B
    # gate, contiguous cache, acceptance from target tokens), else the four calls
    run_step = st.run_fused if st.fused_ok() and not args.separate_calls else st.run
    log(f"warmup {args.warmup} steps")
    for _ in range(args.warmup):
        run_step()
    torch.cuda.synchronize()
    step_fn = run_step
    graph = None
    if args.graph:
        graph = torch.cuda.CUDAGraph()
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            run_step()                    # a warm launch on the capture stream
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        with torch.cuda.graph(graph):
            run_step()
        torch.cuda.synchronize()
        step_fn = graph.replay
        for _ in range(3):
            step_fn()
        torch.cuda.synchronize()

    stream = torch.cuda.current_stream()
    new_ev = lambda: torch.cuda.Event(enable_timing=True)
    flush_k = [0]

    def do_flush():
        if flush is not None:
            flush_k[0] = (flush_k[0] + 1) & 0xFF
            flush.fill_(flush_k[0])
            pkg.echo_probe_stream_read(half[0], half[1], flush_rows, 4, 2, sink)

    def per_step(n, fn, cold):
        """n steps, one event pair around each; with cold, the flush write runs
        between the steps, outside the event pairs.  Returns the step times (ms)."""
        evs = [(new_ev(), new_ev()) for _ in range(n)]
        torch.cuda.synchronize()
        for a, b in evs:
            if cold:
                do_flush()
            a.record(stream)
            fn()
            b.record(stream)
        torch.cuda.synchronize()
        return [a.elapsed_time(b) for a, b in evs]

    cold = flush is not None
    # 1. the timed steps (the contract's K steps): cold unless --flush-mb 0
    log(f"timing {args.steps} {'cold' if cold else 'warm'} steps")
    wall0 = time.perf_counter()
    step_ms = per_step(args.steps, step_fn, cold)
    wall = time.perf_counter() - wall0
    ms_step = float(np.median(step_ms))
    n_proto = max(args.protocol_steps, args.steps)
    proto_ms = step_ms if n_proto == args.steps else per_step(n_proto, step_fn, cold)
    # 2. warm: back-to-back steps between one event pair, and per step
    log(f"timing {n_proto} warm steps")
    ea, eb = new_ev(), new_ev()
    torch.cuda.synchronize()
    ea.record(stream)
    for _ in range(n_proto):
        step_fn()
    eb.record(stream)
    torch.cuda.synchronize()
    warm_mean = ea.elapsed_time(eb) / n_proto
    warm_ms = per_step(n_proto, step_fn, False)
    # 3. the main attention kernel alone: events recorded by the library on its
    # launch stream around that kernel (the timed entry points).  The event
    # packets add idle time around the kernel, so this pass gives the kernel's
    # duration only, not the step time.
    log(f"timing the attention kernel over {n_proto} cold and {n_proto} warm steps")
    kev_c = [(new_ev(), new_ev()) for _ in range(n_proto)]
    kev_w = [(new_ev(), new_ev()) for _ in range(n_proto)]
    # torch reads only an event it has recorded itself: record each once first
    for a, b in kev_c + kev_w:
        a.record(stream)
        b.record(stream)
    torch.cuda.synchronize()
    for evp in kev_c:
        if cold:
            do_flush()
        st.run(attn_events=evp)
    for evp in kev_w:
        st.run(attn_events=evp)
    # the kernel after a write-only flush (dirty lines left in the caches)
    kev_d = [(new_ev(), new_ev()) for _ in range(min(n_proto, 50) if cold else 0)]
    for a, b in kev_d:
        a.record(stream)
        b.record(stream)
    for evp in kev_d:
        flush.fill_(7)
        st.run(attn_events=evp)
    torch.cuda.synchronize()
    kern_c = [a.elapsed_time(b) * 1000.0 for a, b in kev_c]
    kern_w = [a.elapsed_time(b) * 1000.0 for a, b in kev_w]
    kern_d = [a.elapsed_time(b) * 1000.0 for a, b in kev_d]
    attn_us = float(np.mean(kern_c))
    # 4. per-stage times: an event pair around each call of the step, in a pass of
    # its own (the event packets add idle time, so the stages sum to more than a step)
    stages = [("gate", st.gate), ("mask", st.mask), ("attn", st.attn), ("accept", st.accept)]
    if args.serve:
        stages.append(("commit", st.commit))
    n_stage = min(n_proto, 50)
    stage_ev = {name: [] for name, _ in stages}
    torch.cuda.synchronize()
    for _ in range(n_stage):
        if cold:
            do_flush()
        for name, fn in stages:
            a, b = new_ev(), new_ev()
            a.record(stream)
            fn()
            b.record(stream)
            stage_ev[name].append((a, b))
        if args.serve:  # as in a step: the next one repeats this one
            st.cached_len.copy_(st.prefix_len, non_blocking=True)
    torch.cuda.synchronize()
    stage_us = {name: 1000.0 * float(np.median([a.elapsed_time(b) for a, b in evs]))
                for name, evs in stage_ev.items()}
    # 5. the streaming-read ceiling over this batch's own KV cache (both probe
    # modes, each five times after a flush)
    ceiling = {}
    for mode, name in ((0, "plain_loads"), (1, "attention_tile_copies")):
        if mode == 1 and cfg.hkv % 4 != 0:
            continue
        rows_read = st.kv_rows - (st.kv_rows % 32 if mode == 1 else 0)
        ts = []
        for _ in range(5):
            do_flush()
            a, b = new_ev(), new_ev()
            a.record(stream)
            pkg.echo_probe_stream_read(st.k_cache, st.v_cache, rows_read, cfg.hkv, mode, sink)
            b.record(stream)
            torch.cuda.synchronize()
            ts.append(a.elapsed_time(b))
        nbytes = 2 * rows_read * cfg.hkv * cfg.head_dim * 2
        ceiling[name] = nbytes / (float(np.median(ts)) * 1e-3) / 1e9

    res = st.fetch()
    if res["status"] != 0:
        log(f"WARNING: data status bits {res['status']:#x}")
    nq = res["num_slots"]
    value = nq / (ms_step / 1000.0)
    bytes_alg, flops_alg = attn_algorithmic(batch, res, cfg)
    achieved_gbs = bytes_alg / (attn_us * 1e-6) / 1e9
    traffic = traffic_from_profile(attn_source_hash(), {
        "config": args.config, "seed": args.seed, "gate_policy": args.gate_policy,
        "page_size": page_size, "serve": bool(args.serve)})
    kv_bytes = 4 * cfg.hkv * cfg.head_dim * int(batch["prefix_len"].astype(np.int64).sum())
    stats = lambda xs: {"median": float(np.median(xs)), "p10": _pct(xs, 10), "p90": _pct(xs, 90),
                        "mean": float(np.mean(xs)), "n": len(xs)}

    timing_extra = {}
    if kern_d:
        timing_extra["attn_main_us_after_write_only_flush"] = stats(kern_d)
    out = {
        "metric": METRIC,
        "value": value,
        "unit": "verified tree nodes/sec",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_step,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": f"{args.config}: {synth.DESCRIPTION[args.config]}",
            "batch": cfg.R, "budget": cfg.budget, "verified_slots": nq,
            "draft_nodes": int(res["num_selected"]), "candidates": int(batch["cand_offsets"][-1]),
            "kv_prefix_tokens": int(batch["kv_offsets"][-1]), "seed": args.seed,
            "parallelism": "single GPU", "gate_policy": args.gate_policy,
            "checkpoints": checkpoints, "elastic_widths": elastic,
            "kv_layout": f"paged, {page_size}-row pages" if page_size else "contiguous",
            "serve_step": bool(args.serve), "hip_graph": bool(args.graph),
            "entry_point": "echo_verify_step" if run_step == st.run_fused else "four calls",
        },
        "timing": {
            "protocol": (f"value and ms_per_step: median of the {args.steps} timed steps, one "
                         "event pair each" + (f", with {args.flush_mb} MiB written to device "
                                              f"memory and another {args.flush_mb} MiB read "
                                              "between steps (outside the timing)"
                                              if cold else ", back to back")),
            "step_ms_cold" if cold else "step_ms_warm_per_step": stats(proto_ms),
            "step_ms_warm": {"mean_back_to_back": warm_mean, **stats(warm_ms)},
            "attn_main_us_cold" if cold else "attn_main_us": stats(kern_c),
            "attn_main_us_warm": stats(kern_w),
            **timing_extra,
        },
        "roofline": {
            "kernel": "attn_main_kernel",
            "bound": "hbm",
            "achieved": achieved_gbs,
            "peak": PEAK_HBM_GBS,
            "unit": "GB/s",
            "frac": achieved_gbs / PEAK_HBM_GBS,
            "traffic": traffic,
            "algorithmic_bytes": bytes_alg,
            "kernel_us": attn_us,
            "kernel_us_source": ("mean of the cold pass" if cold else "mean") +
                                " (HIP events on the kernel's launch stream)",
            "tflops": flops_alg / (attn_us * 1e-6) / 1e12,
            "mfma_frac": flops_alg / (attn_us * 1e-6) / 1e12 / PEAK_BF16_TFLOPS,
            "read_ceiling_gbs": ceiling,
            "frac_of_read_ceiling": (achieved_gbs / max(ceiling.values())) if ceiling else None,
        },
        "draft_nodes_per_sec": int(res["num_selected"]) / (ms_step / 1000.0),
        "kv_stream_gbs": kv_bytes / (attn_us * 1e-6) / 1e9,
        "stage_us": stage_us,
        "wall_s_timed": wall,
        "mean_accept_len": float(np.mean(res["accept_len"])),
    }
    if cpu is not None:
        out["cpu_baseline"] = cpu
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
