"""Benchmark of one SD^2 speculative-decoding round on one MI355X.

A step is one call of sd2_round: k steered drafter steps, the (k+1)-row verifier
block forward, the accept/resample decision, commit with KV-length rollback and
the steering projection, for every sequence of the batch.  Inputs are synthetic
(seeded N(0, 0.02) weights, uniform-random prompt ids) with the shapes of the
named workload; weights and prompts are resident in HBM before timing starts.

Prints ONE JSON line on stdout; progress goes to stderr.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

import numpy as np  # noqa: E402

PEAK_HBM_GBS = 8000.0


def log(*a):
    print("[bench]", *a, file=sys.stderr, flush=True)


def weight_bytes(dm, esize):
    hd = dm.head_dim
    per_layer = (dm.n_heads * hd + 2 * dm.n_kv_heads * hd) * dm.d_model + dm.d_model * dm.n_heads * hd \
        + 3 * dm.d_ff * dm.d_model
    return (dm.n_layers * per_layer + dm.vocab * dm.d_model) * esize


def kv_row_bytes(dm):
    # K and V of one position across all layers, stored as fp32
    return dm.n_layers * dm.n_kv_heads * dm.head_dim * 2 * 4


def steer_weight_bytes(wl, es, steering="input"):
    """Steering weights read once per round: W_s [d_D][d_V] (input form), or W_hml [d_V][3 d_V]
    plus the per-layer W_s [L_D F_D][d_V] (MLP form)."""
    dV = wl.verifier.d_model
    if steering == "mlp":
        return (3 * dV * dV + wl.drafter.n_layers * wl.drafter.d_ff * dV) * es
    if steering == "mlp-out":
        return (3 * dV * dV + wl.drafter.d_model * dV) * es
    return wl.drafter.d_model * dV * es


def round_bytes(wl, t_avg, steering="input"):
    """Algorithmic HBM bytes of one round for one sequence at round-start length t_avg:
    every weight once per forward (verifier once, drafter k times, steering weights once) plus
    the KV rows each attention pass must read and the rows it appends."""
    es = 2 if wl.dtype == "bf16" else 4
    k = wl.k
    w = weight_bytes(wl.verifier, es) + k * weight_bytes(wl.drafter, es) + steer_weight_bytes(wl, es, steering)
    kv_v = (t_avg + k + (k + 1)) * kv_row_bytes(wl.verifier)
    kv_d = (k * t_avg + k * (k - 1) / 2 + (k + 1)) * kv_row_bytes(wl.drafter)
    return w, kv_v, kv_d


def cpu_baseline(wl, wv, wd, ws, toks, lens, budget_s):
    """The oracle as it stands, on a bounded sample: prefill a short prompt prefix, then time rounds."""
    import oracle

    threads = int(os.environ.get("OMP_NUM_THREADS", os.cpu_count() or 1))
    prefix = min(16, int(lens[0]))
    o = oracle.Oracle(wl, wv, wd, ws, max_batch=1, cap=prefix + wl.new_tokens + wl.k + 1)
    o.prefill_one(0, toks[0, :prefix])
    tokens, rounds, t0 = 0, 0, time.time()
    while time.time() - t0 < budget_s and not o.state(0)["done"]:
        out, lg, _ = o.round_one(0)
        tokens += len(out)
        rounds += 1
        log(f"cpu oracle round {rounds}: {len(out)} tokens, {time.time() - t0:.1f}s")
    dt = time.time() - t0
    return {"value": tokens / dt, "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "sample": f"sequence 0 only, first {prefix} prompt tokens prefilled (untimed), then {rounds} rounds "
                      f"({tokens} tokens) timed; float64 C oracle, OpenMP over output rows"}


# ---------------------------------------------------------------------------------------------
# rocprofv3 post-processing (host-only; no GPU).  Rounds are delimited by k_set_flag, the one
# single-thread kernel every sd2_round launches first.
# ---------------------------------------------------------------------------------------------
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "k_mk_8b-bf16-b1_traffic.json")
TRAFFIC_SOURCES = ("paper_2511_09844_amd/csrc/mk.hip", "paper_2511_09844_amd/csrc/mk.h",
                   "paper_2511_09844_amd/csrc/device_common.h")
ROOFLINE_KERNEL = "k_mk"


def _kclass(name):
    for k in ("k_mk", "k_wsgemv", "k_attn"):
        if k + "(" in name or k + "<" in name:
            return k
    return "other"


def _round_windows(names, skip_first):
    marks = [i for i, n in enumerate(names) if "k_set_flag" in n]
    return list(zip(marks[:-1], marks[1:]))[skip_first:]


def summarize_trace(path, last_eager):
    """Per-round kernel time by class from a kernel_trace.csv: the graph-launched rounds and the
    last `last_eager` (eagerly launched, event-timed) rounds separately."""
    import csv
    rows = []
    with open(path) as f:
        for r in csv.DictReader(f):
            rows.append((int(r["Start_Timestamp"]), int(r["End_Timestamp"]), r["Kernel_Name"]))
    rows.sort()
    wins = _round_windows([r[2] for r in rows], 0)
    groups = (("timed rounds (graph replays; eager launches on the persistent path)", wins[:len(wins) - last_eager]),
              ("profiled (event-timed, eager) rounds", wins[-last_eager:]))
    for title, ws in groups:
        if not ws:
            continue
        per, span = {}, 0
        for a, b in ws:
            span += rows[b][0] - rows[a][0]
            for st, en, n in rows[a:b]:
                c = per.setdefault(_kclass(n), [0, 0])
                c[0] += 1
                c[1] += en - st
        print(f"{title}: {len(ws)} rounds, {span / len(ws) / 1e3:.1f} us per round (first kernel to first kernel)")
        for c, (n, ns) in sorted(per.items(), key=lambda x: -x[1][1]):
            print(f"  {c:9s} {n / len(ws):6.0f} launches/round  {ns / len(ws) / 1e3:9.1f} us/round  "
                  f"avg {ns / n / 1e3:7.2f} us/launch")


def _source_hash():
    import hashlib
    h = hashlib.sha256()
    for p in TRAFFIC_SOURCES:
        with open(os.path.join(ROOT, p), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def summarize_pmc(fetch_csv, write_csv, write_json):
    """HBM traffic per k_mk launch (persistent drafter-step and verify-pass launches) from
    FETCH_SIZE and WRITE_SIZE runs (KiB per dispatch), each scaled by what the same counter reads
    for the 1 GiB calibration copy."""
    import csv
    out = {}
    for counter, path in (("FETCH_SIZE", fetch_csv), ("WRITE_SIZE", write_csv)):
        rows = []
        with open(path) as f:
            for r in csv.DictReader(f):
                rows.append((int(r["Dispatch_Id"]), r["Kernel_Name"], float(r["Counter_Value"])))
        rows.sort()
        wins = _round_windows([r[1] for r in rows], 1)
        n, kib = 0, 0.0
        for a, b in wins:
            for _, name, v in rows[a:b]:
                if _kclass(name) == ROOFLINE_KERNEL:
                    n += 1
                    kib += v
        copy = max((v for _, name, v in rows if "copyBuffer" in name), default=0.0)
        factor = (1 << 20) / copy if copy else float("nan")
        out[counter] = {"launches": n, "kib_per_launch_raw": kib / max(1, n), "copy_kib_raw": copy,
                        "scale": factor, "bytes_per_launch": kib / max(1, n) * factor * 1024}
        print(f"{counter}: {n} {ROOFLINE_KERNEL} launches in {len(wins)} rounds, {kib / max(1, n):.1f} KiB/launch raw; "
              f"1 GiB copy reads {copy:.0f} KiB -> scale {factor:.4f}; {out[counter]['bytes_per_launch'] / 1e6:.3f} MB/launch")
    total = out["FETCH_SIZE"]["bytes_per_launch"] + out["WRITE_SIZE"]["bytes_per_launch"]
    print(f"traffic per {ROOFLINE_KERNEL} launch: {total / 1e6:.3f} MB")
    if write_json:
        rec = {"kernel": ROOFLINE_KERNEL, "workload": "8b-bf16-b1", "source_sha256": _source_hash(),
               "traffic_bytes_per_launch": total, "counters": out}
        with open(write_json, "w") as f:
            json.dump(rec, f, indent=1)
            f.write("\n")


def stored_traffic(workload):
    """Counter-measured bytes per k_mk launch, if taken on the current kernel source and workload."""
    try:
        with open(TRAFFIC_FILE) as f:
            rec = json.load(f)
    except (OSError, ValueError):
        return None
    if rec.get("workload") != workload or rec.get("source_sha256") != _source_hash():
        return None
    return rec.get("traffic_bytes_per_launch")


def main():
    import sd2_inputs as si

    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=30)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default=si.LLAMA8B.name, choices=list(si.BY_NAME))
    ap.add_argument("--prof-rounds", type=int, default=3)
    ap.add_argument("--cpu-budget", type=float, default=20.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--steering", choices=["input", "mlp", "mlp-out"], default="input",
                    help="input: s = W_s h added to the drafter's input embeddings; mlp: the paper's eq. (2) "
                         "per-layer up-projection biases from three verifier layers; mlp-out: its ablation "
                         "with one bias after every drafter MLP (no CPU baseline for either)")
    ap.add_argument("--calib-copy", action="store_true",
                    help="after the rounds, copy one 1 GiB buffer (a plain copy of known size, the reference "
                         "point for scaling hardware traffic counters)")
    ap.add_argument("--summarize-trace", metavar="KERNEL_TRACE_CSV",
                    help="print the per-round breakdown of a rocprofv3 kernel trace of this script and exit")
    ap.add_argument("--summarize-pmc", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="print k_mk HBM traffic from two rocprofv3 --pmc runs of this script with "
                         "--calib-copy and exit")
    ap.add_argument("--write-traffic", action="store_true", help="with --summarize-pmc: store the result")
    args = ap.parse_args()
    if args.summarize_trace:
        summarize_trace(args.summarize_trace, args.prof_rounds)
        return
    if args.summarize_pmc:
        summarize_pmc(*args.summarize_pmc, TRAFFIC_FILE if args.write_traffic else None)
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (the round runs on one device); --gpus {args.gpus} is not supported", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2511_09844_amd import binding as B

    B.load()
    wl = si.BY_NAME[args.workload]
    dev = "cuda:0"
    torch.cuda.set_device(0)
    t0 = time.time()
    keep_host = not args.no_cpu_baseline and args.steering == "input"
    host = {0: {"layers": []}, 1: {"layers": []}}
    models = []
    for which in (0, 1):
        items = []
        for key, arr in si.iter_model_tensors(wl, which):
            items.append((key, arr))
        if keep_host:
            h = host[which]
            for key, arr in items:
                if key[0] == "layers":
                    while len(h["layers"]) <= key[1]:
                        h["layers"].append([])
                    h["layers"][key[1]].append(arr)
                else:
                    h[key[0]] = arr
        models.append(B.DeviceModel(items, dev))
        del items
        log(f"model {which} generated and uploaded ({time.time() - t0:.1f}s)")
    mlp_dev = None
    if args.steering != "input":
        mlp = si.mlp_steer_weights(wl, form=1 if args.steering == "mlp" else 2)
        mlp_dev = {key: B.to_device(mlp[key], dev) for key in ("w_s", "w_hml", "ln_gain", "ln_bias")}
        mlp_dev["ln_eps"] = mlp["ln_eps"]
        del mlp
        ws, ws_dev = None, None
        log(f"MLP steering weights generated and uploaded ({time.time() - t0:.1f}s)")
    else:
        ws = si.steer_weights(wl)
        ws_dev = B.to_device(ws, dev)
    toks, lens = si.prompts(wl)
    stream = torch.cuda.Stream()
    with torch.cuda.stream(stream):
        steer_form = {"input": B.STEER_INPUT, "mlp": B.STEER_MLP, "mlp-out": B.STEER_MLP_OUT}[args.steering]
        eng = B.Engine(B.config_of(wl, steering=steer_form), models[0], models[1], ws_dev, stream=stream,
                       device=dev, mlp=mlp_dev)
        t_tok = torch.from_numpy(toks).to(dev)
        t_len = torch.from_numpy(lens).to(dev)
        torch.cuda.synchronize()
        tp = time.time()
        eng.prefill(t_tok, t_len, wl.max_prompt)
        torch.cuda.synchronize()
        prefill_s = time.time() - tp
        log(f"prefill done in {prefill_s:.2f}s")
        for _ in range(args.warmup):
            eng.round()
        torch.cuda.synchronize()
        st0 = eng.state()
        # one event between consecutive rounds: the whole span gives the mean, the gaps the spread
        evs = [torch.cuda.Event(enable_timing=True) for _ in range(args.steps + 1)]
        evs[0].record(stream)
        for i in range(args.steps):
            eng.round()
            evs[i + 1].record(stream)
        torch.cuda.synchronize()
        ms = evs[0].elapsed_time(evs[-1])
        per_round = sorted(evs[i].elapsed_time(evs[i + 1]) for i in range(args.steps))
        st1 = eng.state()
        log(f"timed {args.steps} rounds: {ms:.2f} ms")
        # kernel-level timing: HIP events around every launch of the same rounds, recorded into the graph
        prof = {c: [0, 0.0, 0.0] for c in (B.PROF_PROGRAM, B.PROF_GEMV, B.PROF_ATTN, B.PROF_SAMPLER, B.PROF_OTHER)}
        stp0 = eng.state()
        if args.prof_rounds > 0:
            eng.profile(True)
            for _ in range(args.prof_rounds):
                eng.round()
                for c in prof:
                    n, pms, pby = eng.profile_read(c)
                    prof[c][0] += n
                    prof[c][1] += pms
                    prof[c][2] += pby
            eng.profile(False)
        torch.cuda.synchronize()
        stp1 = eng.state()
        if args.calib_copy:
            src = torch.empty(1 << 30, dtype=torch.uint8, device=dev).fill_(1)
            dst = torch.empty_like(src)
            torch.cuda.synchronize()
            dst.copy_(src)
            torch.cuda.synchronize()
            del src, dst

    active = [b for b in range(wl.batch) if not st0[b]["done"]]
    tokens = sum(st1[b]["produced"] - st0[b]["produced"] for b in range(wl.batch))
    sec = ms / 1e3
    tau = tokens / (args.steps * max(1, len(active)))
    w_b, kvv_b, kvd_b = 0.0, 0.0, 0.0
    for b in active:
        t_avg = st0[b]["t"] + (st1[b]["t"] - st0[b]["t"]) * (args.steps - 1) / (2 * args.steps)
        w, kvv, kvd = round_bytes(wl, t_avg, args.steering)
        w_b = w
        kvv_b += kvv
        kvd_b += kvd
    bytes_round = w_b + kvv_b + kvd_b
    ms_round = ms / args.steps
    # roofline of the dominant kernel: the persistent launches (weights they stream, from the
    # library, plus the KV rows their attention phases read, from the sequence lengths)
    pr = max(1, args.prof_rounds)
    kv_prof = 0.0
    for b in range(wl.batch):
        if stp0[b]["done"]:
            continue
        t_p = stp0[b]["t"] + (stp1[b]["t"] - stp0[b]["t"]) * (pr - 1) / (2 * pr)
        _, kvv, kvd = round_bytes(wl, t_p)
        kv_prof += (kvv + kvd) * args.prof_rounds
    p_n, p_ms, p_by = prof[B.PROF_PROGRAM]
    if p_n:
        r_kernel = ("k_mk (persistent launch: one per drafter step, one per verify pass; every projection, "
                    "attention and LM head of that forward)")
        g_n, g_ms, g_by = p_n, p_ms, p_by + kv_prof
    else:
        r_kernel = "k_wsgemv (every weight-streaming projection: QKV, O, gate|up, down, LM heads, W_s)"
        g_n, g_ms, g_by = prof[B.PROF_GEMV]
    gemv_gbs = g_by / (g_ms / 1e3) / 1e9 if g_ms > 0 else 0.0
    log(f"round: {ms_round:.3f} ms, {bytes_round / 1e9:.3f} GB algorithmic -> "
        f"{bytes_round / (ms_round / 1e3) / 1e9:.0f} GB/s ({bytes_round / (ms_round / 1e3) / 1e9 / PEAK_HBM_GBS:.1%} of HBM)")
    for c, name in ((B.PROF_PROGRAM, "program"), (B.PROF_GEMV, "gemv"), (B.PROF_ATTN, "attn"),
                    (B.PROF_SAMPLER, "sampler"), (B.PROF_OTHER, "other")):
        n, pms, pby = prof[c]
        log(f"  {name}: {n / max(1, args.prof_rounds):.0f} launches/round, {pms / max(1, args.prof_rounds):.3f} ms/round"
            + (f", {pby / (pms / 1e3) / 1e9:.0f} GB/s" if pby and pms else ""))

    result = {
        "metric": "generated tokens/s at 1 GPU (one SD2 round per step)",
        "value": tokens / sec,
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms_round,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16 weights, f32 activations/KV" if wl.dtype == "bf16" else "f32",
        "data": "synthetic: seeded N(0,0.02) weights, uniform-random prompt ids",
        "config": {"workload": wl.name, "steering": args.steering, "batch": wl.batch, "k": wl.k,
                   "prompt": list(wl.prompt),
                   "new_tokens": wl.new_tokens, "temperature": wl.temperature,
                   "verifier": f"L{wl.verifier.n_layers} d{wl.verifier.d_model} H{wl.verifier.n_heads}/"
                               f"{wl.verifier.n_kv_heads} F{wl.verifier.d_ff} V{wl.verifier.vocab}",
                   "drafter": f"L{wl.drafter.n_layers} d{wl.drafter.d_model} H{wl.drafter.n_heads}/"
                              f"{wl.drafter.n_kv_heads} F{wl.drafter.d_ff}"},
        "round_ms_p50": per_round[len(per_round) // 2],
        "round_ms_p90": per_round[min(len(per_round) - 1, (9 * len(per_round)) // 10)],
        "prefill_s": prefill_s,
        "block_efficiency": tau,
        "round_bytes": bytes_round,
        "round_hbm_frac": bytes_round / (ms_round / 1e3) / 1e9 / PEAK_HBM_GBS,
        "roofline": {"bound": "hbm", "kernel": r_kernel,
                     "achieved": gemv_gbs, "peak": PEAK_HBM_GBS, "unit": "GB/s", "frac": gemv_gbs / PEAK_HBM_GBS,
                     "traffic": stored_traffic(wl.name) if p_n and args.steering == "input" else None,
                     "launches_per_round": g_n / max(1, args.prof_rounds),
                     "avg_launch_us": g_ms / max(1, g_n) * 1e3,
                     "bytes_per_launch": g_by / max(1, g_n)},
        "cpu_baseline": None,
    }
    if not args.no_cpu_baseline and args.steering == "input":
        result["cpu_baseline"] = cpu_baseline(wl, host[0], host[1], ws, toks, lens, args.cpu_budget)
    eng.close()
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
