"""Benchmark of the DFlow round on one MI355X.

A step is one speculative round over the batch: dflow_draft_block (relay +
drafter), forced-draft construction, dflow_verify_block, dflow_accept_and_carry
and kv_commit.  The drafter runs in full every round; the block sent to
verification is forced from the target's own greedy trajectory with a seeded
geometric acceptance schedule, because a random-init drafter accepts almost
nothing.  The trajectory is produced beforehand on the GPU by junk-draft
rounds through the same kernels.  Inputs (weights, KV cache, trajectory,
schedule) are resident in HBM before the timed region starts.

With --temperature T > 0 a step is the sampling-decoding round instead
(drafts drawn from the drafter, speculative-sampling acceptance), with no
forcing.

Prints one JSON line: committed tokens/s and ms per round, the dominant
kernel's HBM roofline (live HIP-event timing, HBM traffic from the recorded
counter pass) and the CPU oracle timed on a bounded sample of the workload.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "committed tokens/s + ms/round, Qwen3-8B-shape B=16; % HBM roofline"
HBM_PEAK_GBS = 8000.0
MFMA_PEAK_TFLOPS = {"bf16": 2500.0, "f32": 157.3}   # dense matrix-core peaks of the MI355X
ROLLOUT_GAMMA = 7.0   # decay of the rollout loss over draft positions


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=128)
    ap.add_argument("--warmup", type=int, default=8)
    ap.add_argument("--workload", default="qwen3-8b")
    ap.add_argument("--carry", choices=["on", "off"], default="on")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-kernel-timing", action="store_true")
    ap.add_argument("--cpu-sample-ctx", type=int, default=48,
                    help="prompt tokens of the oracle rollout sample (--rollout); greedy and sampled rounds are "
                         "timed at the workload's own context")
    ap.add_argument("--batch", type=int, default=0, help="override the workload's sequence count (batch sweeps)")
    ap.add_argument("--prefill-rows", type=int, default=512,
                    help="prompt rows per prefill chunk (the library's max_rows; set-up only, the rounds are unchanged)")
    ap.add_argument("--rollout", type=int, default=0,
                    help="k > 0: time forward-only multi-round rollouts (a mask round and k relay rounds, "
                         "transitions on the target's greedy trajectory); a step is one rollout")
    ap.add_argument("--temperature", type=float, default=0.0,
                    help="T > 0: sampling decoding (speculative sampling, the drafter's own samples) instead of "
                         "greedy rounds with forced acceptance")
    ap.add_argument("--eager", action="store_true",
                    help="issue the greedy round's launches one by one instead of replaying its recorded HIP graph")
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="run one device-to-device copy of this size first (calibrates HBM counters)")
    ap.add_argument("--counter-pass", action="store_true",
                    help="the program of an HBM counter pass (run under rocprofv3 --pmc): set-up prefill, the "
                         "calibration copy, then --steps eager rounds with the drafter's own drafts; no timing, "
                         "no JSON line")
    ap.add_argument("--traffic-record", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="write the dominant kernel's HBM counter record from the counter_collection.csv files of "
                         "a FETCH_SIZE and a WRITE_SIZE counter pass (host only, no GPU)")
    return ap.parse_args()


TRAFFIC_FILE = os.path.join(ROOT, "profiles", "traffic.json")
# the dominant kernel at the Qwen3-8B shape: the gate|up SwiGLU projection of a round (M = 16 rows)
TRAFFIC_KERNEL = ("gemm.swiglu N=24576 K=4096 M=16", "_ZN5dflow11gemm_kernelINS_4bf16ELi2ELi1ELi3ELb1EEEvNS_10GemmParamsE",
                  "gemm_kernel<dflow::bf16, 2, 1, 3, true>", 24576 * 4096 * 2 + 16 * 4096 * 2 + 16 * 12288 * 2)
COPY_KERNEL = "__amd_rocclr_copyBuffer"
PROF_EVENTS = 16384   # launches the library's per-launch event record holds (dflow_profile)
NSEG = 4   # timed segments (median and min per-step time besides the whole-run value)


def measured_traffic(kernel_name):
    """HBM bytes per launch of the dominant kernel from the committed counter
    record (FETCH_SIZE + WRITE_SIZE, each scaled by the same counter's reading
    for a copy of known size), or None when the record is absent, is for
    another kernel, or the kernel's machine code in the loaded library differs
    from the code the counters were taken on (the record's measured_on digest
    when it has one: the code that actually ran under the counters)."""
    from paper_2609_06498_amd import library_path
    from paper_2609_06498_amd.codeobj import kernel_code_digest
    try:
        with open(TRAFFIC_FILE) as fh:
            rec = json.load(fh)
        measured = (rec.get("measured_on") or {}).get("code_sha256", rec.get("code_sha256"))
        if rec.get("kernel") != kernel_name or \
                measured != kernel_code_digest(library_path(), rec.get("symbol", "")):
            return None
    except (OSError, ValueError, KeyError):
        return None
    return int(rec["fetch_bytes"] + rec["write_bytes"])


def profiled_steps(steps, rounds_per_step, gemm_launches, attn_layers):
    """Steps of the per-launch event pass: about 64 rounds, at most `steps`,
    and no more than the library's event record holds (PROF_EVENTS launches:
    the step's GEMM launches plus one attention launch per layer and round)."""
    per_step = gemm_launches + attn_layers * rounds_per_step
    return max(1, min(steps, 64 // rounds_per_step, PROF_EVENTS // per_step))


def write_traffic_record(fetch_csv, write_csv, copy_mib=256):
    """HBM bytes per launch of the dominant kernel from two rocprofv3 counter
    passes of `bench.py --counter-pass --calib-copy-mib 256`: each counter's
    mean per dispatch of that kernel, divided by the same counter's reading
    per byte of the calibration copy (copy_mib MiB read and written).  The
    record is keyed to the kernel's machine code in the library built here."""
    import csv
    from paper_2609_06498_amd import library_path
    from paper_2609_06498_amd.codeobj import kernel_code_digest
    name, symbol, pretty, alg = TRAFFIC_KERNEL
    copy_bytes = copy_mib << 20

    def read(path, counter):
        per, copies = [], []
        with open(path) as fh:
            for r in csv.DictReader(fh):
                if r["Counter_Name"] != counter:
                    continue
                v = float(r["Counter_Value"])
                if pretty in r["Kernel_Name"]:
                    per.append(v)
                elif COPY_KERNEL in r["Kernel_Name"]:
                    copies.append(v)
        if not per or not copies:
            raise SystemExit(f"{path}: no {counter} records for {pretty} or the calibration copy")
        return sum(per) / len(per), max(copies), len(per)

    f_kib, f_copy, nd = read(fetch_csv, "FETCH_SIZE")
    w_kib, w_copy, _ = read(write_csv, "WRITE_SIZE")
    ff, wf = f_copy * 1024 / copy_bytes, w_copy * 1024 / copy_bytes
    rec = {"kernel": name, "symbol": symbol, "code_sha256": kernel_code_digest(library_path(), symbol),
           "fetch_bytes": int(round(f_kib * 1024 / ff)), "write_bytes": int(round(w_kib * 1024 / wf)),
           "fetch_kib_per_dispatch": round(f_kib, 1), "write_kib_per_dispatch": round(w_kib, 1), "dispatches": nd,
           "calibration_copy_bytes": copy_bytes, "copy_fetch_kib": f_copy, "copy_write_kib": w_copy,
           "fetch_factor": round(ff, 5), "write_factor": round(wf, 5), "algorithmic_bytes": alg}
    with open(TRAFFIC_FILE, "w") as fh:
        json.dump(rec, fh, indent=1)
        fh.write("\n")
    print(json.dumps(rec))


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


def gemm_bytes(rt, nseq, verify_lm_head=True, relay=True):
    """Algorithmic bytes of every weight-streaming GEMM launch of one round:
    each weight byte once, the A operand once, the output once.  A rollout
    round verifies without the LM head; a round without relay runs no relay
    MLP."""
    dm, B = rt.dims, rt.block
    elt = 2 if dm.dtype == "bf16" else 4
    M = nseq * B
    d, F, V, qd, kvd = dm.d, dm.ffn, dm.vocab, dm.q_dim, dm.kv_dim
    qkv = qd + 2 * kvd

    def g(N, K, out_elt=elt, n_out=None):
        return N * K * elt + M * K * elt + M * (N if n_out is None else n_out) * out_elt

    # the QKV projection writes its fp32 partial sums, one per K part
    layer = g(qkv, d, 4 * rt.qkv_parts) + g(d, qd) + g(2 * F, d, n_out=F) + g(d, F)
    verify = dm.n_layers * layer + (g(V, d, 0) if verify_lm_head else 0)
    draft = dm.n_draft_layers * layer + g(V, d, 0) + ((g(dm.d_h, 3 * d) + g(2 * d, dm.d_h, 4)) if relay else 0)
    accept = g(d, dm.m * d, 4)
    commit = g(dm.n_draft_layers * 2 * kvd, d)   # the drafter layers' context K/V in one GEMM
    launches = (dm.n_layers + dm.n_draft_layers) * 4 + (2 if verify_lm_head else 1) + (2 if relay else 0) + 1 + 1
    return verify + draft + accept + commit, launches


def attention_bytes(rt, start_pos, n_layers):
    """Algorithmic bytes of the attention launches of one round over n_layers
    layers: every visible key and value once (t_s context positions plus the
    B block rows of each sequence), the block's queries once and the
    attention output once.  start_pos: host [b] anchor positions t_s."""
    dm, B = rt.dims, rt.block
    elt = 2 if dm.dtype == "bf16" else 4
    per_layer = sum((int(t) + B) * 2 * dm.kv_dim * elt + 2 * B * dm.q_dim * elt for t in start_pos)
    return n_layers * per_layer


def measured_stream_peaks():
    """Streaming rates of plain library kernels on this device, for context
    next to the published peak: a 1 GiB device copy (read + write bytes) and
    a 2 GiB fp32 sum (read bytes), each the best of 5 timed runs."""
    import torch
    out = {}
    n = (1 << 30) // 4
    src = torch.ones(2 * n, dtype=torch.float32, device="cuda")
    dst = torch.empty(n, dtype=torch.float32, device="cuda")
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)

    def best(fn, nbytes):
        fn()
        torch.cuda.synchronize()
        t = []
        for _ in range(5):
            e0.record()
            fn()
            e1.record()
            torch.cuda.synchronize()
            t.append(e0.elapsed_time(e1) * 1e-3)
        return round(nbytes / min(t) / 1e9, 1)

    out["copy_GB_s"] = best(lambda: dst.copy_(src[:n]), 2 * n * 4)
    out["sum_read_GB_s"] = best(lambda: src.sum(), 2 * n * 4)
    del src, dst
    torch.cuda.empty_cache()
    return out


def build_trajectory(rt, sess, prompts, need, sched, B, b):
    """Target trajectory T*: the greedy continuation of every prompt, made by
    junk-draft rounds through the same kernels (each commits at least the
    bonus token).  Returns (traj [b, L] device, L, mode, tok) for forcing."""
    import torch
    t = time.time()
    sess.prefill(prompts)
    torch.cuda.synchronize()
    P = [len(p) for p in prompts]
    first_anchor = sess.anchor.clone()
    L = max(need)
    traj = torch.zeros(b, L, dtype=torch.int32, device="cuda")
    for s in range(b):
        traj[s, :P[s]] = torch.from_numpy(prompts[s]).cuda()
    zmode = torch.zeros(b, B, dtype=torch.int8, device="cuda")
    ztok = torch.zeros(b, B, dtype=torch.int32, device="cuda")
    hist_com, hist_acc, hist_pos = [], [], []
    done = 0
    while done < max(n - p for n, p in zip(need, P)):
        pos = sess.seq_len.clone()
        rt.force_drafts(b, traj, 1, zmode, ztok, sess.anchor, sess.seq_len, sess.block)
        rt.verify_block(b, sess.block, sess.seq_len, sess.tgt)
        rt.accept_and_carry(b, sess.block, sess.tgt, sess.accept, sess.anchor, sess.committed, sess.n_carry)
        rt.kv_commit(b, sess.accept, sess.seq_len)
        hist_com.append(sess.committed.clone())
        hist_acc.append(sess.accept.clone())
        hist_pos.append(pos)
        if len(hist_com) % 8 == 0:
            done = int((sess.seq_len.cpu().numpy() - np.array(P)).min())
    torch.cuda.synchronize()
    traj_h = np.zeros((b, L), np.int32)
    fa = first_anchor.cpu().numpy()
    for s in range(b):
        traj_h[s, :P[s]] = prompts[s]
        traj_h[s, P[s]] = fa[s]
    for com, acc, pos in zip(hist_com, hist_acc, hist_pos):
        com, acc, pos = com.cpu().numpy(), acc.cpu().numpy(), pos.cpu().numpy()
        for s in range(b):
            for j in range(acc[s] + 1):
                p = pos[s] + 1 + j
                if p < L:
                    traj_h[s, p] = com[s, j]
    traj.copy_(torch.from_numpy(traj_h))
    log(f"trajectory ({len(hist_com)} junk rounds) in {time.time() - t:.1f}s")
    assert rt.status() == 0
    return traj, L, torch.from_numpy(sched["mode"]).cuda(), torch.from_numpy(sched["tok"]).cuda()


def main():
    args = parse()
    if args.traffic_record:
        write_traffic_record(*args.traffic_record, copy_mib=args.calib_copy_mib or 256)
        return
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (got --gpus {args.gpus}): the DFlow round is a single-GPU "
              f"data-parallel step (sequences shard across GPUs with no exchange); it runs on one GPU only.", file=sys.stderr)
        sys.exit(2)
    import torch
    from paper_2609_06498_amd import Runtime
    from paper_2609_06498_amd.session import Session
    from workload import get_config
    from workload.synth import make_prompts, make_schedule, make_weights, trajectory_length_needed

    wl = get_config(args.workload)
    if args.batch > 0:
        wl = wl.with_(batch=args.batch)
    dm, B, b = wl.dims, wl.block, wl.batch
    K = args.steps
    log(f"workload {wl.name}: {wl.description}; steps {K} warmup {args.warmup}")
    t = time.time()
    w = make_weights(dm, wl.seed_w)
    log(f"weights generated in {time.time() - t:.1f}s")
    prompts = make_prompts(wl)
    sched = make_schedule(wl, max(K, args.warmup))
    need = trajectory_length_needed(wl, sched)
    # the junk-draft trajectory rounds advance every sequence together until the
    # longest continuation is done (checked every 8 rounds, <= B tokens each)
    P0 = [len(p) for p in prompts]
    max_ctx = max(P0) + max(n - p for n, p in zip(need, P0)) + 9 * B
    sampled = args.temperature > 0
    kr = args.rollout
    if sampled and kr > 0:
        print("--temperature and --rollout are exclusive", file=sys.stderr)
        sys.exit(2)
    if sampled:   # every timed phase restarts from the prompts and commits at most B tokens per round
        max_ctx = max(P0) + (max(K, args.warmup) + 2) * B
    if kr > 0:    # rollout rounds advance a + 1 tokens along the trajectory; random drafts match it rarely
        roll_rounds = max(K, args.warmup) * (kr + 1)
        need = [p + 2 * roll_rounds + 2 * B for p in P0]
        max_ctx = max(need) + 10 * B
    t = time.time()
    rt = Runtime(dm, B, b, max_ctx, w, wl.carry_window, max_rows=args.prefill_rows)
    torch.cuda.synchronize()
    log(f"runtime created (upload + pack) in {time.time() - t:.1f}s")
    if args.no_cpu_baseline:
        del w
    sess = Session(rt, b)
    if args.calib_copy_mib > 0:   # a plain copy of known size, for the HBM counter calibration
        n = args.calib_copy_mib << 20
        src = torch.ones(n // 4, dtype=torch.float32, device="cuda")
        dst = torch.empty_like(src)
        dst.copy_(src)
        torch.cuda.synchronize()
        log(f"calibration copy: {n} bytes read, {n} bytes written")
        del src, dst

    carry_on = args.carry == "on"
    if args.counter_pass:   # the rounds' kernels with the drafter's own drafts, nothing timed
        sess.prefill(prompts)
        for _ in range(K):
            sess.round(carry_on)
        torch.cuda.synchronize()
        log(f"counter pass: {K} rounds, status {rt.status()}")
        return
    if kr > 0:
        traj, L, _, _ = build_trajectory(rt, sess, prompts, need, sched, B, b)

        def reset():
            sess.prefill(prompts)   # the prefill's anchor is the trajectory's token after the prompt

        def run(n, r0=0):
            for r in range(r0, r0 + n):
                sess.rollout(traj, L, kr, ROLLOUT_GAMMA, carry_on)
        run_eager = run
    elif sampled:
        streams = torch.arange(b, dtype=torch.int64, device="cuda")
        smp = rt.sampler(args.temperature, 1234, streams)

        def reset():
            sess.prefill(prompts)

        def run(n, r0=0):
            for r in range(r0, r0 + n):
                sess.round_sampled(smp, carry_on)
        run_eager = run
    else:
        traj, L, mode_d, tok_d = build_trajectory(rt, sess, prompts, need, sched, B, b)

        def reset():
            sess.prefill(prompts)

        def run_eager(n, r0=0):
            for r in range(r0, r0 + n):
                sess.round(carry_on, force=(traj, L, mode_d[r], tok_d[r]))

        run = run_eager
        if not args.eager:   # the round as one recorded HIP graph, replayed with each round's forcing plan
            reset()
            run_eager(1)      # first launches (launch-attribute set-up) outside the capture
            replay = sess.capture_round(carry_on, force=(traj, L))

            def run(n, r0=0):
                for r in range(r0, r0 + n):
                    replay(mode_d[r], tok_d[r])

    reset()
    run(args.warmup)
    torch.cuda.synchronize()
    t_pre = time.perf_counter()   # the prompts' prefill (set-up, outside the timed rounds)
    reset()
    torch.cuda.synchronize()
    t_pre = time.perf_counter() - t_pre
    n_pre = int(sum(len(p) for p in prompts))
    log(f"prefill of {n_pre} prompt tokens: {t_pre * 1e3:.1f} ms ({n_pre / t_pre:.0f} tokens/s, "
        f"{args.prefill_rows}-row chunks)")
    len0 = sess.seq_len.cpu().numpy().copy()
    # the K timed steps in NSEG consecutive segments, each bracketed by HIP
    # events on the round stream (no synchronisation inside the timed region)
    nseg = NSEG if K % NSEG == 0 and K >= 2 * NSEG else 1
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(nseg + 1)]
    t0 = time.perf_counter()
    ev[0].record()
    for i in range(nseg):
        run(K // nseg, i * K // nseg)
        ev[i + 1].record()
    torch.cuda.synchronize()
    dt = time.perf_counter() - t0
    seg_ms = [ev[i].elapsed_time(ev[i + 1]) / (K // nseg) for i in range(nseg)]
    len1 = sess.seq_len.cpu().numpy()
    committed = int((len1 - len0).sum())
    expect = None if (sampled or kr > 0) else int((sched["accept"][:K] + 1).sum())
    diverged = expect is not None and committed != expect
    status = rt.status()
    tau_cfg = None
    if not sampled and kr == 0 and wl.schedule == "geometric":   # E[min(G, K)] + 1 of the forcing law
        q = wl.sched_param / (1.0 + wl.sched_param)
        tau_cfg = round(1.0 + sum(min(k, wl.K) * (1 - q) * q ** k for k in range(4000)), 4)
    tok_s = committed / dt
    ms_round = dt * 1e3 / K
    rounds_per_step = kr + 1 if kr > 0 else 1
    tau = committed / (K * b * rounds_per_step)
    if kr > 0:
        assert int(len1.max()) + B <= L, "the rollouts ran past the trajectory"
    log(f"timed {K} {'rollouts' if kr > 0 else 'rounds'}: {ms_round:.3f} ms/step, {tok_s:.1f} tok/s, "
        f"tau {tau:.3f} per round "
        + (f"(sampling T={args.temperature})" if sampled else
           f"(rollout k={kr}, {ms_round / rounds_per_step:.3f} ms/round)" if kr > 0 else
           f"(schedule {expect / (K * b):.3f})")
        + f", status {status}; {nseg} segments: median {np.median(seg_ms):.3f}, min {min(seg_ms):.3f} ms/step")

    # ---- live per-kernel timing with HIP events on the round's stream
    roofline, kernels = None, None
    if kr > 0:   # per rollout: the mask round, then k relay rounds, all verifying without the LM head
        g0, n0 = gemm_bytes(rt, b, verify_lm_head=False, relay=False)
        g1, n1 = gemm_bytes(rt, b, verify_lm_head=False, relay=carry_on)
        gb, nl = g0 + kr * g1, n0 + kr * n1
    else:
        gb, nl = gemm_bytes(rt, b, relay=carry_on)
    if not args.no_kernel_timing:
        kp = profiled_steps(K, rounds_per_step, nl, dm.n_layers + dm.n_draft_layers)
        reset()
        torch.cuda.synchronize()
        rt.profile(True)
        pos_hist = []
        for r in range(kp):   # the anchor positions of every round (device copies; no synchronisation)
            pos_hist.append(sess.seq_len.clone())
            run_eager(1, r)
        torch.cuda.synchronize()
        entries = rt.profile_read()
        rt.profile(False)
        pos_hist = [p.cpu().numpy() for p in pos_hist]
        # attention: algorithmic bytes from the host-known positions (the library records 0)
        attn_bytes = {"verify": sum(attention_bytes(rt, p, dm.n_layers) for p in pos_hist),
                      "draft": sum(attention_bytes(rt, p, dm.n_draft_layers) for p in pos_hist)}
        for e in entries:
            if e["name"] == "attention" and e["phase"] in attn_bytes:
                e["bytes"] = attn_bytes[e["phase"]]
        gemms = [e for e in entries if e["name"].startswith("gemm")]
        assert sum(e["launches"] for e in gemms) == kp * nl, (entries, kp, nl)
        lib_bytes = sum(e["bytes"] for e in gemms)
        assert abs(lib_bytes - kp * gb) <= 1e-6 * kp * gb, (lib_bytes, kp * gb)
        kernels = []
        for e in sorted(entries, key=lambda e: -e["ms"]):
            avg_us = e["ms"] * 1e3 / e["launches"]
            k = {"kernel": e["name"], "phase": e["phase"], "N": e["N"], "K": e["K"], "M": e["M"],
                 "per_round": e["launches"] / kp, "avg_us": round(avg_us, 3), "ms_per_round": round(e["ms"] / kp, 4)}
            if e["bytes"]:
                k["GB_s"] = round(e["bytes"] / e["launches"] / (avg_us * 1e-6) / 1e9, 1)
            if e["name"].startswith("gemm"):   # matrix-core rate: 2 M N K flops per launch
                k["TFLOP_s"] = round(2.0 * e["M"] * e["N"] * e["K"] / (avg_us * 1e-6) / 1e12, 2)
            kernels.append(k)
        dom = max(gemms, key=lambda e: e["ms"])
        avg_s = dom["ms"] * 1e-3 / dom["launches"]
        per_launch = dom["bytes"] / dom["launches"]
        achieved = per_launch / avg_s / 1e9
        fam_ms = sum(e["ms"] for e in gemms)
        kname = f"{dom['name']} N={dom['N']} K={dom['K']} M={dom['M']}"
        roofline = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                    "frac": round(achieved / HBM_PEAK_GBS, 4), "traffic": measured_traffic(kname),
                    "kernel": kname,
                    "algorithmic_bytes_per_launch": int(per_launch), "avg_launch_us": round(avg_s * 1e6, 3),
                    "gemm_family_GB_s": round(lib_bytes / (fam_ms * 1e-3) / 1e9, 1),
                    "gemm_family_ms_per_round": round(fam_ms / kp, 4)}
        tflops = 2.0 * dom["M"] * dom["N"] * dom["K"] / avg_s / 1e12     # the secondary (matrix-core) bound
        roofline["mfma_TFLOP_s"] = round(tflops, 2)
        roofline["mfma_frac"] = round(tflops / MFMA_PEAK_TFLOPS[dm.dtype], 4)
        peaks = measured_stream_peaks()
        roofline["measured_stream_GB_s"] = peaks
        roofline["frac_of_measured_copy"] = round(achieved / peaks["copy_GB_s"], 4)

        def path(sel):   # algorithmic bytes over the summed live kernel time of the selected launches
            es = [e for e in entries if sel(e)]
            nb, ms = sum(e["bytes"] for e in es), sum(e["ms"] for e in es)
            if ms <= 0:
                return None
            gbs = nb / (ms * 1e-3) / 1e9
            return {"GB_per_round": round(nb / kp / 1e9, 4), "ms_per_round": round(ms / kp, 4),
                    "GB_s": round(gbs, 1), "frac": round(gbs / HBM_PEAK_GBS, 4)}

        # the verify path of the round (its GEMMs, attention and LM head), the
        # verify attention alone, and the drafter's forward
        roofline["verify_path"] = path(lambda e: e["phase"] == "verify")
        roofline["verify_gemms"] = path(lambda e: e["phase"] == "verify" and e["name"].startswith("gemm"))
        roofline["verify_attention"] = path(lambda e: e["phase"] == "verify" and e["name"] == "attention")
        roofline["draft_path"] = path(lambda e: e["phase"] == "draft")
        round_gb = sum(e["bytes"] for e in entries) / kp
        roofline["round"] = {"GB_per_round": round(round_gb / 1e9, 4),
                             "GB_s_at_ms_per_step": round(round_gb / (ms_round * 1e-3) / 1e9, 1),
                             "frac": round(round_gb / (ms_round * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)}
        log(f"verify path {roofline['verify_path']}; verify attention {roofline['verify_attention']}; "
            f"round {roofline['round']}")
        log(f"stream rates on this device: {peaks}")
        log(f"dominant {roofline['kernel']}: avg {avg_s * 1e6:.2f} us, {achieved:.1f} GB/s; "
            f"gemm family {roofline['gemm_family_GB_s']} GB/s, {fam_ms / kp:.3f} ms/round")
        for k in kernels:
            log(f"  {k}")

    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(wl, w, prompts, tau, args.cpu_sample_ctx, args.temperature, kr)

    out = {"metric": METRIC, "value": round(tok_s, 2), "unit": "tokens/s", "n_gpus": 1, "steps": K,
           "warmup": args.warmup, "ms_per_step": round(ms_round, 4), "higher_is_better": True, "scaling": "weak",
           "vs_baseline": None, "dtype": "bf16" if dm.dtype == "bf16" else "f32",
           "data": ("synthetic (seeded random-init weights, uniform prompts, speculative sampling at "
                    f"T={args.temperature} with the drafter's own samples)") if sampled else
                   ("synthetic (seeded random-init weights, uniform prompts, forward-only rollouts on the "
                    "target's greedy trajectory with the drafter's own proposals)") if kr > 0 else
                   "synthetic (seeded random-init weights, uniform prompts, forced geometric acceptance)",
           "config": {"workload": wl.name, "batch": b, "block": B, "ctx": list(wl.ctx), "rounds": K,
                      "carry": args.carry,
                      "schedule": f"sampling T={args.temperature}" if sampled else
                      f"rollout k={kr}, gamma {ROLLOUT_GAMMA}" if kr > 0 else f"{wl.schedule}({wl.sched_param})",
                      "tau_realised": round(tau, 4), "tau_configured": tau_cfg,
                      "tokens_per_s_at_configured_tau": (round(tau_cfg * b / (ms_round * 1e-3), 2)
                                                         if tau_cfg is not None else None),
                      "trajectory_diverged": diverged, "status": status,
                      "launch": "eager" if (args.eager or sampled or kr > 0) else "hip_graph",
                      "parallelism": "single GPU"},
           "prefill": {"tokens": n_pre, "chunk_rows": args.prefill_rows, "ms": round(t_pre * 1e3, 2),
                       "tokens_per_s": round(n_pre / t_pre, 1)},
           "segments_ms_per_step": {"n": nseg, "each": [round(x, 4) for x in seg_ms],
                                    "median": round(float(np.median(seg_ms)), 4), "min": round(min(seg_ms), 4)},
           "roofline": roofline, "cpu_baseline": cpu, "kernels": kernels}
    print(json.dumps(out), flush=True)


def synthetic_oracle_state(o, prompt, anchor, seed=7):
    """An oracle sequence state at the prompt's full length whose caches (target
    K/V, fused features, drafter context K/V) hold seeded random values of the
    right sizes.  A round's cost depends only on these sizes, and the oracle
    cannot prefill thousands of tokens within a benchmark's time; the values
    are for timing only and are never compared with anything."""
    dm = o.m.dims
    dt = o.m.mode.dt
    t = len(prompt)
    g = np.random.default_rng(seed)
    kv = lambda: (g.random((t, dm.n_kv_heads, dm.head_dim), dtype=np.float32) - 0.5).astype(dt)
    st = o.empty_state()
    st.k = [kv() for _ in range(dm.n_layers)]
    st.v = [kv() for _ in range(dm.n_layers)]
    st.F = (g.random((t, dm.d), dtype=np.float32) - 0.5).astype(dt)
    st.ck = [kv() for _ in range(dm.n_draft_layers)]
    st.cv = [kv() for _ in range(dm.n_draft_layers)]
    st.tokens = [int(x) for x in prompt] + [int(anchor)]
    return st


def cpu_baseline(wl, w, prompts, tau, ctx_len, temperature=0.0, rollout_k=0):
    """The oracle timed on this host on a bounded sample of the workload: one
    sequence at its full context length (the first prompt's), one untimed
    round (it converts the weights and leaves a carry record), then the mean
    of two timed rounds (draft + verify + accept + commit, or their sampled
    form at T > 0); tokens/s = the GPU run's realised tau per sequence / the
    oracle's round time.  A rollout sample prefills ctx_len tokens instead."""
    from oracle import Mode, OracleDFlow, OracleModel
    dm = wl.dims
    mode = "bf16" if dm.dtype == "bf16" else "fp32"
    m = OracleModel(dm, w, Mode(mode), cache=True)
    o = OracleDFlow(m, wl.block, wl.carry_window)
    rng = np.random.default_rng(0)
    n_rounds = 2
    if rollout_k > 0:   # one rollout of k + 1 rounds on a random trajectory (its cost does not depend on the tokens)
        import oracle.rollout as ro
        p = prompts[0][:ctx_len]
        traj = np.concatenate([p, rng.integers(0, dm.vocab, (rollout_k + 1) * wl.block + 2)])
        st = ro.anchor_state(o, traj, len(p))
        t = time.perf_counter()
        ro.rollout(o, st, traj, rollout_k, ROLLOUT_GAMMA)
        t_round = (time.perf_counter() - t) / (rollout_k + 1)
        n_rounds, ctx = rollout_k + 1, len(p)
    else:
        p = prompts[0]
        ctx = len(p)
        s = synthetic_oracle_state(o, p, int(rng.integers(0, dm.vocab)))
        blk = lambda: np.concatenate([[s.anchor], rng.integers(0, dm.vocab, wl.K)])

        def one():
            if temperature > 0:
                o.round_sampled(s, temperature, 1234, 0, True)
            else:
                o.round(s, True, block=blk())
        one()   # untimed: weight conversion, carry record
        t = time.perf_counter()
        for _ in range(n_rounds):
            one()
        t_round = (time.perf_counter() - t) / n_rounds
    try:
        import threadpoolctl
        info = threadpoolctl.threadpool_info()
        threads = max([i.get("num_threads", 1) for i in info] or [1])
    except Exception:
        threads = os.cpu_count()
    log(f"oracle: {n_rounds} rounds at context {ctx}, {t_round:.2f}s each, {threads} BLAS threads")
    return {"value": round(tau / t_round, 4), "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "ctx": ctx,
            "sample": f"mean of {n_rounds} {mode} oracle rounds (draft+verify+accept+commit, relay on"
                      + (f", speculative sampling T={temperature}" if temperature > 0 else "")
                      + (f", one forward-only rollout k={rollout_k} after a {ctx}-token prefill" if rollout_k > 0
                         else f", one sequence at its full {ctx}-position context, caches of seeded random "
                              f"values") + f") of {wl.name}; tokens/s = GPU-realised tau {tau:.3f} per sequence / "
                      f"{t_round:.2f} s; host cpu_count {os.cpu_count()}"}


if __name__ == "__main__":
    main()
