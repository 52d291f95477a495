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
    """sha256 of what the attention kernel is built from: its source and the build
    script (which holds its compiler flags)."""
    h = hashlib.sha256()
    for rel in (("paper_2604_09603_amd", "csrc", "attn.hip"), ("paper_2604_09603_amd", "build.py")):
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


def cpu_baseline(batch, cfg, checkpoints=None, elastic=None, budget_s=12.0):
    """The oracle as written, single-threaded, on a bounded sample of the workload."""
    import numpy as np
    from threadpoolctl import threadpool_limits

    import oracle
    import synth
    with threadpool_limits(limits=1):
        t0 = time.perf_counter()
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
        t_front = time.perf_counter() - t0
        qo = m["q_offsets"]
        P = batch["prefix_len"].astype(np.int64)
        n = np.diff(qo)
        work_all = float((P * n).sum())
        order = np.random.default_rng(0).permutation(cfg.R)
        done_work, t_attn, used = 0.0, 0.0, []
        for r in order:
            rows = list(range(int(qo[r]), int(qo[r + 1])))
            t1 = time.perf_counter()
            oracle.tree_verify_attn(batch["q"], batch["k_new"], batch["v_new"], batch["k_cache"],
                                    batch["v_cache"], batch["kv_offsets"], qo, m["tree_mask"],
                                    cfg.hq, cfg.hkv, batch["sm_scale"], rows=rows)
            t_attn += time.perf_counter() - t1
            done_work += float(P[r] * n[r])
            used.append(int(r))
            if t_front + t_attn >= budget_s:
                break
    nq = int(qo[-1])
    est = t_front + t_attn * work_all / max(done_work, 1.0)
    return {
        "value": nq / est, "unit": "verified tree nodes/sec", "cores": 1, "kind": "oracle",
        "sample": (f"oracle gate+mask+accept on the full batch ({t_front:.2f} s) and float64 "
                   f"attention for {len(used)} of {cfg.R} requests ({t_attn:.2f} s, "
                   f"{100.0 * done_work / work_all:.1f}% of the prefix-key work), attention time "
                   f"scaled by prefix-key work to the whole step ({est:.1f} s)"),
    }


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=50)
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--config", default="q235b")
    ap.add_argument("--seed", type=int, default=3)
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
    ap.add_argument("--graph", action="store_true",
                    help="capture one step in a HIP graph and time graph replays")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="BYTES",
                    help="only run a plain device-to-device copy of BYTES, five times (the "
                         "reference kernel that scales the HBM byte counters)")
    args = ap.parse_args()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (asked for --gpus {args.gpus}): the verification "
              "step runs on a single MI355X and there is no multi-GPU path.", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    if args.copy_calibration > 0:
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
    import paper_2604_09603_amd as pkg
    from paper_2604_09603_amd.step import VerifyStep

    cfg = synth.CONFIGS[args.config]
    log(f"generating {args.config} seed={args.seed}")
    t0 = time.time()
    batch = synth.make_batch(args.config, args.seed)
    log(f"generated in {time.time() - t0:.1f} s; uploading")
    elastic = None
    if args.gate_policy == "elastic":
        checkpoints = gate_checkpoints("sparse", args.config, cfg.depth)
        elastic = (2, cfg.branch)
    else:
        checkpoints = gate_checkpoints(args.gate_policy, args.config, cfg.depth)
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
    torch.cuda.synchronize()

    log(f"warmup {args.warmup} steps")
    for _ in range(args.warmup):
        st.run()
    torch.cuda.synchronize()
    step_fn = st.run
    if args.graph:
        graph = torch.cuda.CUDAGraph()
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            st.run()                      # a warm launch on the capture stream
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        with torch.cuda.graph(graph):
            st.run()
        torch.cuda.synchronize()
        step_fn = graph.replay
        for _ in range(3):
            step_fn()
        torch.cuda.synchronize()

    stream = torch.cuda.current_stream()
    # 1. the timed steps: the whole step, nothing else on the stream
    t_start = torch.cuda.Event(enable_timing=True)
    t_end = torch.cuda.Event(enable_timing=True)
    log(f"timing {args.steps} steps")
    torch.cuda.synchronize()
    wall0 = time.perf_counter()
    t_start.record(stream)
    for _ in range(args.steps):
        step_fn()
    t_end.record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - wall0
    ms_total = t_start.elapsed_time(t_end)
    ms_step = ms_total / args.steps
    # 2. the same steps again with HIP events around the main attention kernel,
    # recorded by the library on its launch stream.  The event packets add a few
    # microseconds of idle time around that kernel, so this pass gives the
    # kernel's duration only, not the step time.
    ev_a = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    ev_b = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps)]
    # torch only reads an event it has recorded itself: record each once, the library re-records
    for e in ev_a + ev_b:
        e.record(stream)
    log(f"timing the attention kernel over {args.steps} steps")
    torch.cuda.synchronize()
    for i in range(args.steps):
        pkg.set_attn_profile_events(ev_a[i], ev_b[i])
        st.run()
    torch.cuda.synchronize()
    pkg.set_attn_profile_events(None, None)
    attn_ms = [a.elapsed_time(b) for a, b in zip(ev_a, ev_b)]
    attn_us = 1000.0 * float(np.mean(attn_ms))
    # 3. per-stage times: an event pair around each call of the step, in a pass of
    # its own (the event packets add idle time, so the stages sum to more than a step)
    stages = [("gate", st.gate), ("mask", st.mask), ("attn", st.attn), ("accept", st.accept)]
    if args.serve:
        stages.append(("commit", st.commit))
    n_stage = min(args.steps, 20)
    stage_ev = {name: [] for name, _ in stages}
    torch.cuda.synchronize()
    for _ in range(n_stage):
        for name, fn in stages:
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(stream)
            fn()
            b.record(stream)
            stage_ev[name].append((a, b))
        if args.serve:  # as in a step: the next one repeats this one
            st.cached_len.copy_(st.prefix_len, non_blocking=True)
    torch.cuda.synchronize()
    stage_us = {name: 1000.0 * float(np.mean([a.elapsed_time(b) for a, b in evs]))
                for name, evs in stage_ev.items()}

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
            "tflops": flops_alg / (attn_us * 1e-6) / 1e12,
            "mfma_frac": flops_alg / (attn_us * 1e-6) / 1e12 / PEAK_BF16_TFLOPS,
        },
        "draft_nodes_per_sec": int(res["num_selected"]) / (ms_step / 1000.0),
        "kv_stream_gbs": 4 * cfg.hkv * cfg.head_dim * int(batch["prefix_len"].astype(np.int64).sum())
                         / (attn_us * 1e-6) / 1e9,
        "stage_us": stage_us,
        "wall_s_timed": wall,
        "mean_accept_len": float(np.mean(res["accept_len"])),
    }
    if not args.no_cpu_baseline:
        log("timing the CPU oracle on a bounded sample")
        out["cpu_baseline"] = cpu_baseline(batch, cfg, checkpoints, elastic)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
