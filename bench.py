#!/usr/bin/env python3
"""Benchmark of DVI's self-speculative decode step on one MI355X.

A step is one pass of the whole hot path for every sequence of the batch: k_spec serial
drafts through layers 1..k plus the LoRA draft head, one block verify through layers
k+1..L plus the frozen head, the commit (longest agreeing prefix, KV rollback, replay
logging) and, on workloads that train the drafter, the periodic drafter update.  The
prompt is prefilled before timing; weights, KV cache and prompt are resident in HBM.

Prints ONE JSON line: committed tokens/s of the whole job (value), ms per step, the
verify-step and draft-token HBM bandwidth from HIP events, the roofline of the dominant
kernel (its algorithmic bytes per launch over its HIP-event duration), acceptance
statistics, the same engine decoding plainly (k_spec = 1) for the speedup ratio, and the
CPU oracle timed on the host cores on a bounded sample of the same workload.

Usage: python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload 7b] [--k-spec 4]
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0     # MI355X HBM3E, published
METRIC = "committed tokens/s (7B shape, bs=1) + verify-step HBM GB/s vs peak"
PAPER_CONTEXT = ("paper: 2.16x average wall-time speedup over greedy AR decoding on 1x NVIDIA H100 "
                 "(Vicuna-7B, Spec-Bench, split k=2, k_spec=4); no absolute tokens/s published")
KERNEL_NAMES = {"gate_up": "gemm_kernel<bf16,MG=1,EPI_SWIGLU> (gate/up projection, SwiGLU epilogue)",
                "qkv": "gemm_kernel<bf16,MG=1,EPI_QKV>", "down": "gemm_kernel<bf16,MG=1,EPI_RESID> (MLP down)",
                "head": "gemm_kernel<bf16,MG=1,EPI_LOGITS>",
                "attention": "attn_kernel<bf16,128> (split-KV MFMA attention with in-kernel merge)"}


# Measured HBM traffic of a probed kernel: the committed summary of two rocprofv3 --pmc passes
# (FETCH_SIZE, WRITE_SIZE) over this benchmark, scaled by what the same counters read for a
# plain device copy.  Used only while the kernel source it was taken on is unchanged.
TRAFFIC_PROFILES = {"gate_up": "profiles/gemm_gate_up_7b_b1_k4_traffic.md"}
# the device code of every kernel: a counter summary stands only while these are unchanged
KERNEL_SOURCES = ("paper_2510_05421_amd/csrc/kernels.hip", "paper_2510_05421_amd/csrc/device.h")


def kernel_sources_sha256():
    """SHA-256 over the kernel sources, in the order listed."""
    import hashlib
    h = hashlib.sha256()
    for rel in KERNEL_SOURCES:
        with open(os.path.join(ROOT, rel), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def profile_fields(rel):
    """The `- `key`: `value`` fields of a committed counter summary, or {} when it is missing or
    was taken on other kernel sources than the current ones."""
    if rel is None or not os.path.exists(os.path.join(ROOT, rel)):
        return {}
    fields = {}
    with open(os.path.join(ROOT, rel)) as f:
        for line in f:
            if line.startswith("- `") and "`: " in line:
                key, val = line[3:].split("`: ", 1)
                fields[key] = val.strip().strip("`")
    return fields if fields.get("kernel_sources_sha256") == kernel_sources_sha256() else {}


def measured_traffic(probe, workload, k_spec):
    """Bytes per launch from the committed counter summary, or None when there is none for
    this kernel and workload or the kernel source has changed since it was taken."""
    fields = profile_fields(TRAFFIC_PROFILES.get(probe))
    if fields.get("workload") != workload or fields.get("k_spec") != str(k_spec):
        return None
    return int(float(fields["traffic_bytes_per_launch"]))


# MFMA counters of the drafter update's forward GEMM over a full replay ring: the committed
# summary of a rocprofv3 --pmc pass (SQ_INSTS_VALU_MFMA_MOPS_BF16, SQ_VALU_MFMA_BUSY_CYCLES,
# GRBM_GUI_ACTIVE) over this benchmark's 13B workload.
MFMA_PROFILE = "profiles/drafter_update_13b.md"


def measured_mfma(workload):
    fields = profile_fields(MFMA_PROFILE)
    if fields.get("workload") != workload:
        return None
    return {"forward_gemm_counter_gflop": float(fields["forward_gemm_counter_gflop"]),
            "forward_gemm_counter_tflop_s": float(fields["forward_gemm_counter_tflop_s"]),
            "forward_gemm_mfma_frac_of_peak": float(fields["forward_gemm_mfma_frac_of_peak"]),
            "forward_gemm_mfma_busy_frac": float(fields["forward_gemm_mfma_busy_frac"]),
            "source": MFMA_PROFILE}


def log(msg):
    print("[bench] " + msg, file=sys.stderr, flush=True)


def algorithmic_bytes(shape, layers, rows_per_seq, lens, head_rows, lora=False):
    """Bytes a pass must move: each weight once, keys/values read over the context and
    written for the new rows, the head logits written.  rows_per_seq tokens per sequence."""
    es = 2 if shape.bf16 else 4
    w = layers * shape.layer_params() * es + shape.vocab * shape.d_model * es
    if lora:
        w += shape.vocab * shape.lora_rank * 4 + shape.lora_rank * shape.d_model * 4
    kv = 0
    for L0 in lens:
        kv += layers * (L0 + rows_per_seq) * shape.kv_dim * 2 * es   # read 0..len+rows-1 (incl. new)
    return w + kv + head_rows * shape.vocab * 4


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--workload", default="7b")
    ap.add_argument("--no-ceiling", action="store_true",
                    help="skip the full-acceptance leg (drafts forced to the greedy continuation)")
    ap.add_argument("--k-spec", type=int, default=None)
    ap.add_argument("--probe", default="gate_up", choices=sorted(KERNEL_NAMES))
    ap.add_argument("--probe-steps", type=int, default=20)
    ap.add_argument("--ar-steps", type=int, default=40)
    ap.add_argument("--cpu-seconds", type=float, default=20.0,
                    help="decode time of the CPU oracle leg after its full prefill (at least --cpu-steps steps)")
    ap.add_argument("--cpu-steps", type=int, default=8)
    ap.add_argument("--read-rate-mib", type=int, default=2048,
                    help="buffer of the streaming-read reference (the measured HBM ceiling); 0 skips it")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-ar", action="store_true")
    ap.add_argument("--no-full-update", action="store_true",
                    help="skip timing the drafter update over a full replay ring")
    ap.add_argument("--no-device-steps", action="store_true",
                    help="skip the leg that runs the decode loop through dvi_decode_steps")
    ap.add_argument("--copy-calib-mib", type=int, default=0,
                    help="first run 3 plain device-to-device copies of this many MiB (a reference for "
                         "the hardware byte counters under a profiler)")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: the decode step runs on a single MI355X "
              "(there is no multi-GPU path); run with --gpus 1", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch
    import synth
    from paper_2510_05421_amd.engine import Engine, EngineConfig

    if args.copy_calib_mib > 0:
        n = args.copy_calib_mib << 20
        src = torch.empty(n, dtype=torch.uint8, device="cuda:0").fill_(1)
        dst = torch.empty_like(src)
        for _ in range(3):
            dst.copy_(src)
        torch.cuda.synchronize()
        log("copy calibration: 3 device copies of %d bytes" % n)
        del src, dst

    wl = synth.WORKLOADS[args.workload]
    shape = wl.model
    k = args.k_spec or wl.k_spec[0]
    B, P, N = wl.batch, wl.prompt_len, wl.new_tokens
    W = args.warmup
    K = args.steps if args.steps is not None else max(1, min(100, (N - 1) // k - W))
    if (W + K) * k >= N:
        sys.exit("warmup+steps (%d) x k_spec (%d) exceeds the workload's %d new tokens" % (W + K, k, N))

    log("workload %s: generating weights" % wl.name)
    t = time.time()
    w = synth.make_weights(shape, 0)
    prompts = synth.make_prompts(shape.vocab, B, P, 0)
    log("weights ready in %.1f s; building engine" % (time.time() - t))
    cfg = EngineConfig.from_shape(shape, max_batch=B, max_seq=P + N + 2 * k + 2, max_k_spec=max(k, 8),
                                  buffer_rows=wl.buffer_rows)
    eng = Engine(cfg, w, "cuda:0")
    # the practical HBM read ceiling: the decode GEMMs' streaming loads over a buffer far larger than
    # the 256 MB last-level cache, fastest of five passes
    peak_meas = None
    if args.read_rate_mib > 0:
        peak_meas = eng.read_rate(args.read_rate_mib << 20, reps=5)
        log("streaming-read reference: %.0f GB/s over %d MiB (%.3f of the nominal %g)"
            % (peak_meas, args.read_rate_mib, peak_meas / HBM_PEAK_GBS, HBM_PEAK_GBS))
    from paper_2510_05421_amd.schedule import KLRLSchedule
    sched = KLRLSchedule()

    remaining = np.full(B, N - 1, np.int32)
    state = {"step": 0}

    def update_drafter(stats=None):
        c = sched.coeffs(eng.updates, eng.baseline)
        st = eng.update_drafter(c["c_kl"], c["c_ce"], c["c_pg"], c["c_ent"], c["tau"], eng.baseline, lr=1e-3)
        if st["fresh"] > 0:
            eng.baseline = sched.ema(eng.baseline, st["fresh_accepted"] / st["fresh"])
        eng.updates += 1
        if stats is not None:
            stats["update_ms"].append(eng.timings()["update"])
            stats["update_rows"].append(st["rows"])

    def step(kk, stats=None, update=True, forced=None):
        lens_before = eng_lens[:]
        eng.draft(kk, forced=forced)
        eng.verify()
        tok, n, m = eng.commit(max_new=remaining)
        remaining[:] = remaining - n
        for b in range(B):
            eng_lens[b] += int(n[b])
        state["step"] += 1
        if update and wl.update_every and kk > 1 and state["step"] % wl.update_every == 0:
            update_drafter(stats)
        if stats is not None:
            tm = eng.timings()
            stats["tokens"] += int(n.sum())
            stats["m"].append(m.copy())
            stats["n"].append(n.copy())
            stats["verify_ms"].append(tm["verify"])
            stats["draft_ms"].append(tm["draft"])
            stats["verify_bytes"].append(algorithmic_bytes(shape, shape.n_layers - shape.split_k, kk,
                                                           lens_before, B * kk))
            stats["draft_bytes"].append(sum(algorithmic_bytes(shape, shape.split_k, 1,
                                                              [l0 + j for l0 in lens_before], B, lora=True)
                                            for j in range(kk)))

    log("prefill %d x %d tokens" % (B, P))
    t = time.time()
    eng.prefill(prompts)
    torch.cuda.synchronize()
    pf_s = time.time() - t
    # dense work of the prefill: every layer's matrices on every prompt token (+ the head on the
    # last token of each sequence); attention adds about 2 * P * d * L per token on top
    pf_flop = 2.0 * B * P * shape.layer_params() * shape.n_layers + 2.0 * B * shape.vocab * shape.d_model
    prefill = {"s": round(pf_s, 4), "tokens": B * P, "gemm_tflop": round(pf_flop / 1e12, 2),
               "tflop_s": round(pf_flop / pf_s / 1e12, 1)}
    log("prefill %.2f s (%.1f TFLOP of GEMM work, %.0f TFLOP/s)" % (pf_s, pf_flop / 1e12, pf_flop / pf_s / 1e12))
    eng_lens = [P] * B
    for _ in range(W):
        step(k)
    st = {"tokens": 0, "m": [], "n": [], "verify_ms": [], "draft_ms": [], "verify_bytes": [], "draft_bytes": [],
          "update_ms": [], "update_rows": []}
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for _ in range(K):
        step(k, st)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    elapsed = t1 - t0
    value = st["tokens"] / elapsed
    ms_step = 1e3 * elapsed / K
    mv = np.array(st["m"])
    nv = np.array(st["n"])
    ver_ms = float(np.median(st["verify_ms"]))
    ver_gbs = float(np.mean(st["verify_bytes"])) / (ver_ms * 1e-3) / 1e9
    dr_ms = float(np.median(st["draft_ms"]))
    dr_gbs = float(np.mean(st["draft_bytes"])) / (dr_ms * 1e-3) / 1e9
    step_bytes = float(np.mean(st["draft_bytes"])) + float(np.mean(st["verify_bytes"]))
    step_gbs = step_bytes / (ms_step * 1e-3) / 1e9
    log("timed %d steps: %.1f tokens/s, %.2f ms/step, mean m %.2f, verify %.3f ms (%.0f GB/s), "
        "draft %.3f ms (%.0f GB/s)" % (K, value, ms_step, mv.mean(), ver_ms, ver_gbs, dr_ms, dr_gbs))
    # drafter update (the workloads that train the drafter): its dense work is the LoRA head
    # forward over the ring, rows x V x (d + r) multiply-adds, plus the gradient products
    upd = None
    if st["update_ms"]:
        u_ms = float(np.median(st["update_ms"]))
        rows = int(np.median(st["update_rows"]))
        V, d, r = shape.vocab, shape.d_model, shape.lora_rank
        flops = 2.0 * rows * V * (d + r) + 2.0 * (V * r * rows + rows * V * r + r * d * rows)
        tfs = flops / (u_ms * 1e-3) / 1e12
        peak = 2500.0 if shape.bf16 else 157.3
        upd = {"updates": len(st["update_ms"]), "ms": round(u_ms, 4), "rows": rows, "gflop": round(flops / 1e9, 2),
               "tflop_s": round(tfs, 2), "mfma_peak_tflop_s": peak, "frac": round(tfs / peak, 4),
               "head_bytes": shape.vocab * shape.d_model * (2 if shape.bf16 else 4)}
        log("drafter update: %d updates, median %.3f ms over %d rows: %.1f GFLOP -> %.1f TFLOP/s (%.3f of %g)"
            % (len(st["update_ms"]), u_ms, rows, flops / 1e9, tfs, tfs / peak, peak))

    # the drafter update over a full ring (the workload's 256-row buffer): random-weight trajectories
    # accept too few drafts to fill it within the timed window, so its rows are synthetic here
    upd_full = None
    if wl.update_every and not args.no_full_update:
        R = wl.buffer_rows
        buf = synth.make_buffer(shape.d_model, shape.vocab, R, seed=11)
        eng.write_buffer(buf.h, buf.a, buf.logits, buf.r, buf.fresh)
        c = sched.coeffs(eng.updates, eng.baseline)
        times = []
        for _ in range(6):
            eng.update_drafter(c["c_kl"], c["c_ce"], c["c_pg"], c["c_ent"], c["tau"], eng.baseline, lr=0.0)
            times.append(eng.timings()["update"])
        u_ms = float(np.median(times[1:]))
        V, d, r = shape.vocab, shape.d_model, shape.lora_rank
        flops = 2.0 * R * V * (d + r) + 2.0 * (V * r * R + R * V * r + r * d * R)
        gemm_flops = 2.0 * R * V * d
        peak = 2500.0 if shape.bf16 else 157.3
        upd_full = {"rows": R, "ms": round(u_ms, 4), "gflop": round(flops / 1e9, 2),
                    "tflop_s": round(flops / (u_ms * 1e-3) / 1e12, 2), "mfma_peak_tflop_s": peak,
                    "frac": round(flops / (u_ms * 1e-3) / 1e12 / peak, 4), "forward_gemm_gflop": round(gemm_flops / 1e9, 2),
                    # matrix-unit utilisation of the forward GEMM read from rocprofv3 counters
                    "mfma_counters": measured_mfma(wl.name)}
        log("drafter update over a full %d-row ring: %.3f ms, %.1f GFLOP -> %.1f TFLOP/s (%.3f of %g)"
            % (R, u_ms, flops / 1e9, upd_full["tflop_s"], upd_full["frac"], peak))

    # dominant kernel: every launch of one kernel class timed with HIP events on the engine's stream
    # (a sequence that has all its tokens keeps computing with its commits masked, so the
    # kernel sees the same shapes whether or not the probe pass runs past the last token)
    roof = None
    if args.probe_steps > 0:
        eng.probe(args.probe)
        for _ in range(args.probe_steps):
            step(k, update=False)
        pr = eng.probe_read()
        eng.probe("off")
        if pr["launches"]:
            avg_ms = pr["ms"] / pr["launches"]
            per_launch = pr["bytes"] / pr["launches"]
            achieved = per_launch / (avg_ms * 1e-3) / 1e9
            roof = {"bound": "hbm", "achieved": round(achieved, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                    "frac": round(achieved / HBM_PEAK_GBS, 4),
                    "peak_measured": round(peak_meas, 1) if peak_meas else None,
                    "frac_of_measured": round(achieved / peak_meas, 4) if peak_meas else None,
                    # the step the metric names: the whole verify pass against the same peaks
                    "verify_step_frac": round(ver_gbs / HBM_PEAK_GBS, 4),
                    "verify_step_frac_of_measured": round(ver_gbs / peak_meas, 4) if peak_meas else None,
                    "traffic": measured_traffic(args.probe, wl.name, k),
                    "kernel": KERNEL_NAMES[args.probe], "launches": pr["launches"],
                    "avg_us": round(avg_ms * 1e3, 2), "bytes_per_launch": int(per_launch)}
            log("probe %s: %d launches, avg %.1f us, %.0f GB/s" % (args.probe, pr["launches"], avg_ms * 1e3,
                                                                  achieved))

    ar = None
    if not args.no_ar:
        eng.prefill(prompts)
        remaining[:] = N - 1
        eng_lens[:] = [P] * B
        for _ in range(W):
            step(1)
        sa = {"tokens": 0, "m": [], "n": [], "verify_ms": [], "draft_ms": [], "verify_bytes": [], "draft_bytes": [],
              "update_ms": [], "update_rows": []}
        KA = min(args.ar_steps, N - 1 - W)
        torch.cuda.synchronize()
        a0 = time.perf_counter()
        for _ in range(KA):
            step(1, sa)
        torch.cuda.synchronize()
        a1 = time.perf_counter()
        ar_tps = sa["tokens"] / (a1 - a0)
        ar = {"tokens_per_s": round(ar_tps, 2), "steps": KA, "speedup": round(value / ar_tps, 3)}
        log("plain AR on the same engine: %.1f tokens/s -> speedup %.2fx" % (ar_tps, value / ar_tps))
    # The same decode loop through dvi_decode_steps: several steps per call, queued without a host
    # synchronisation between them (the drafter update, where the workload trains, between calls).
    dev = None
    if not args.no_device_steps:
        per_call = wl.update_every if (wl.update_every and k > 1) else 16
        eng.prefill(prompts)
        left = np.full(B, N - 1, np.int32)
        _, n0, _ = eng.decode_steps(k, max(1, min(W, 64)), max_new=left)
        left = left - n0.sum(axis=0)
        calls = max(1, K // per_call)
        dtok, dms = 0, []
        torch.cuda.synchronize()
        d0 = time.perf_counter()
        for _ in range(calls):
            _, n1, m1 = eng.decode_steps(k, per_call, max_new=left)
            left = left - n1.sum(axis=0)
            dtok += int(n1.sum())
            dms.append(m1)
            if wl.update_every and k > 1:
                update_drafter()
        torch.cuda.synchronize()
        d1 = time.perf_counter()
        dev_tps = dtok / (d1 - d0)
        dev = {"tokens_per_s": round(dev_tps, 2), "steps": calls * per_call, "steps_per_call": per_call,
               "ms_per_step": round(1e3 * (d1 - d0) / (calls * per_call), 4),
               "mean_m": round(float(np.concatenate(dms).mean()), 4)}
        log("dvi_decode_steps, %d steps per call: %.1f tokens/s, %.2f ms/step, mean m %.2f"
            % (per_call, dev_tps, dev["ms_per_step"], dev["mean_m"]))
    # Full-acceptance ceiling: the same step with every draft forced to the verifier's own greedy
    # continuation (taken from a plain-decoding run), so each step commits k_spec tokens.  The
    # drafter head still runs in full (its argmax is replaced afterwards); no drafter updates.
    ceil = None
    if not args.no_ceiling:
        NG = (W + K) * k + 1
        greedy, _ = eng.generate(prompts, NG, 1)
        eng.prefill(prompts)
        remaining[:] = N - 1
        eng_lens[:] = [P] * B
        for s_ in range(W):
            step(k, update=False, forced=greedy[:, s_ * k + 1:s_ * k + k + 1])
        sc = {"tokens": 0, "m": [], "n": [], "verify_ms": [], "draft_ms": [], "verify_bytes": [], "draft_bytes": [],
              "update_ms": [], "update_rows": []}
        torch.cuda.synchronize()
        c0 = time.perf_counter()
        for s_ in range(W, W + K):
            step(k, sc, update=False, forced=greedy[:, s_ * k + 1:s_ * k + k + 1])
        torch.cuda.synchronize()
        c1 = time.perf_counter()
        mc = np.array(sc["m"])
        ceil_tps = sc["tokens"] / (c1 - c0)
        ceil = {"tokens_per_s": round(ceil_tps, 2), "steps": K, "ms_per_step": round(1e3 * (c1 - c0) / K, 4),
                "mean_m": round(float(mc.mean()), 4), "tokens_per_step": round(sc["tokens"] / (K * B), 4),
                "verify_ms": round(float(np.median(sc["verify_ms"])), 4),
                "draft_ms": round(float(np.median(sc["draft_ms"])), 4),
                "speedup_vs_ar": round(ceil_tps / ar["tokens_per_s"], 3) if ar else None}
        log("full-acceptance ceiling (drafts forced to the greedy continuation): %.1f tokens/s, mean m %.2f, "
            "%.2f ms/step%s" % (ceil_tps, mc.mean(), ceil["ms_per_step"],
                                 " -> %.2fx plain AR" % ceil["speedup_vs_ar"] if ar else ""))
    eng.close()
    del eng

    cpu = None
    if not args.no_cpu_baseline:
        import oracle
        from oracle import dvi as odvi
        cores = int(os.environ.get("OMP_NUM_THREADS", len(os.sched_getaffinity(0))))
        om = oracle.OracleModel(w)
        drafter = odvi.Drafter(w.lora_A.astype(np.float64), w.lora_B.astype(np.float64), shape.lora_gamma)
        # the workload itself on sequence 0: the full prompt prefilled, then decode steps at that
        # context -- at least cpu_steps, and as many as fit in about cpu_seconds after the first
        marks = {}
        steps_cap = max(args.cpu_steps, 1)

        class _Enough(Exception):
            pass

        def on_step(res, s_):
            marks.setdefault("steps", []).append(time.perf_counter())
            marks["committed"] = len(res.tokens) - 1     # tokens after the prefill's first one
            if s_ + 1 >= steps_cap and marks["steps"][-1] - marks["prefill"] > args.cpu_seconds:
                raise _Enough

        c0 = time.perf_counter()
        try:
            odvi.dvi_generate(om, prompts[0], N, k, drafter, max_steps=N,
                              on_prefill=lambda: marks.__setitem__("prefill", time.perf_counter()),
                              on_step=on_step)
        except _Enough:
            pass
        steps_done, committed = len(marks["steps"]), marks["committed"]
        pre_s = marks["prefill"] - c0
        dec_s = marks["steps"][-1] - marks["prefill"]
        cpu = {"value": round(committed / dec_s, 4), "unit": "tokens/s", "cores": cores, "kind": "oracle",
               "prefill_s": round(pre_s, 2),
               "sample": "float64 oracle DVI rollout (k_spec=%d) of the same model on sequence 0 of the workload: "
                         "its full %d-token prompt prefilled in %.1f s (not in the rate), then %d decode steps "
                         "at that context, %d committed tokens in %.1f s" % (k, P, pre_s, steps_done, committed,
                                                                             dec_s)}
        log("cpu oracle: %s" % cpu["sample"])

    dt = "bf16" if shape.bf16 else "f32"
    out = {
        "metric": METRIC, "value": round(value, 3), "unit": "tokens/s", "n_gpus": 1, "steps": K, "warmup": W,
        "ms_per_step": round(ms_step, 4), "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": dt, "data": "synthetic",
        "config": {"workload": "%s: %dL split k=%d, d=%d, %dx%d heads (%d kv), SwiGLU %d, vocab %d, %s; "
                               "batch %d, %d-token random prompt, %d new tokens, k_spec=%d"
                               % (wl.name, shape.n_layers, shape.split_k, shape.d_model, shape.n_heads,
                                  shape.head_dim, shape.n_kv_heads, shape.ffn_dim, shape.vocab, dt, B, P, N, k),
                   "batch": B, "prompt_len": P, "new_tokens": N, "k_spec": k, "split_k": shape.split_k},
        "roofline": roof,
        "cpu_baseline": cpu,
        "verify_step": {"ms": round(ver_ms, 4), "gb_s": round(ver_gbs, 1), "frac": round(ver_gbs / HBM_PEAK_GBS, 4),
                        "bytes": int(np.mean(st["verify_bytes"]))},
        "draft_token": {"ms": round(dr_ms / k, 4), "gb_s": round(dr_gbs, 1), "frac": round(dr_gbs / HBM_PEAK_GBS, 4)},
        # the whole step (k_spec draft passes + verify, wall time of the timed loop): its frac is
        # also committed tokens/s over the rate the same bytes would allow at the HBM peak
        "step": {"ms": round(ms_step, 4), "bytes": int(step_bytes), "gb_s": round(step_gbs, 1),
                 "frac": round(step_gbs / HBM_PEAK_GBS, 4),
                 "tokens_per_s_at_peak": round(float(nv.mean()) * B / (step_bytes / (HBM_PEAK_GBS * 1e9)), 1)},
        "acceptance": {"mean_m": round(float(mv.mean()), 4), "mean_tokens_per_step": round(float(nv.mean()), 4),
                       "rate": round(float(mv.mean()) / k, 4)},
        "ar_baseline": ar,
        "full_acceptance": ceil,
        "device_steps": dev,
        "prefill": prefill,
        "drafter_update": upd,
        "drafter_update_full_ring": upd_full,
        "paper_context": PAPER_CONTEXT,
    }
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
