"""Benchmark of SD^2 speculative decoding on one MI355X.

A step is one whole generation of the named workload: sd2_prefill of the prompts,
then sd2_round until every sequence has its new tokens.  Each round is k steered
drafter steps, the (k+1)-row verifier block forward, the accept/resample
decision, commit with KV-length rollback and the steering projection, for every
sequence of the batch.  The first warm-up generation reads the state after every
round to learn how many rounds a generation takes; generations are deterministic
(fixed Philox stream, fixed reduction orders), so the timed ones replay exactly
those rounds with no host synchronisation.  Events between rounds give per-round
latency; bytes per round are counted at each round's own context length.

Inputs are synthetic (seeded N(0, 0.02) weights, uniform-random prompt ids) with
the shapes of the named workload; weights and prompts are resident in HBM before
timing starts.  Prints ONE JSON line on stdout; progress goes to stderr.
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
    return {"value": tokens / dt, "unit": "tokens/s", "cores": threads, "kind": "oracle", "cpu": cpu_model(),
            "sample": f"sequence 0 only, first {prefix} prompt tokens prefilled (untimed), then {rounds} rounds "
                      f"({tokens} tokens) timed; float64 C oracle, OpenMP over output rows (the round's cost is "
                      f"its weights: KV reads at a {prefix}-token context instead of 512-768 change it by about 2 %)"}


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


def _trace_rows(path):
    """(kernel name, start ns, end ns) of every dispatch in a rocprofv3 kernel trace: the rocpd
    database (`*_results.db`, the default output) or a kernel_trace.csv."""
    if path.endswith(".db"):
        import sqlite3
        con = sqlite3.connect(path)
        rows = list(con.execute("select name, start, end from kernels order by start"))
        con.close()
        return rows
    import csv
    with open(path) as f:
        return sorted(((r["Kernel_Name"], int(r["Start_Timestamp"]), int(r["End_Timestamp"]))
                       for r in csv.DictReader(f)), key=lambda x: x[1])


def summarize_trace(path):
    """Per-kernel launches and time from a rocprofv3 kernel trace of this script, rounds apart from
    the rest: a round runs from k_set_flag (its first kernel) to k_commit (its last); every other
    launch (prefill, set-up) is listed in a second table."""
    per = {True: {}, False: {}}
    rounds, in_round = 0, False
    for name, start, end in _trace_rows(path):
        if "k_set_flag" in name:
            rounds += 1
            in_round = True
        key = name.split("(")[0].replace("void ", "").replace("sd2::", "")
        c = per[in_round].setdefault(key, [0, 0])
        c[0] += 1
        c[1] += end - start
        if "k_commit" in name:
            in_round = False
    for inside, title in ((True, f"{rounds} rounds in the trace; kernels inside rounds"),
                          (False, "kernels outside rounds (prefill, set-up)")):
        tab = per[inside]
        tot = sum(v[1] for v in tab.values())
        print(f"{title}: {tot / 1e6:.2f} ms" + (f", {tot / 1e6 / max(1, rounds):.3f} ms/round" if inside else ""))
        for key, (n, ns) in sorted(tab.items(), key=lambda x: -x[1][1])[:20]:
            print(f"  {key[:40]:40s} {n:7d} launches {n / max(1, rounds):6.2f}/round  {ns / 1e6:10.2f} ms total  "
                  f"avg {ns / n / 1e3:9.2f} us")
    mk = [v for k, v in per[True].items() if k.startswith("k_mk<")]
    if mk:
        n, ns = sum(v[0] for v in mk), sum(v[1] for v in mk)
        print(f"k_mk, all instances: {n} launches, average {ns / n / 1e3:.2f} us")


def _source_hash():
    import hashlib
    h = hashlib.sha256()
    for p in TRAFFIC_SOURCES:
        with open(os.path.join(ROOT, p), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def summarize_stages(path, k):
    """Per-round kernel time of a rocprofv3 kernel trace of this script, split by stage of the
    round: drafter step 1, drafter steps 2..k (each ends with its k_pick_final), the verify pass
    (up to the accept test) and the sampling and commit kernels after it."""
    stages = ["drafter step 1", f"drafter steps 2-{k}", "verify pass", "accept, commit"]
    per = [dict() for _ in stages]
    rounds, st = 0, None
    for name, start, end in _trace_rows(path):
        key = name.split("(")[0].replace("void ", "").replace("sd2::", "")
        if "k_set_flag" in key:
            rounds, st, picks = rounds + 1, 0, 0
        if st is None:
            continue
        if key.startswith("k_row_partial") or key.startswith("k_accept"):
            st = 3
        c = per[st].setdefault(key, [0, 0])
        c[0] += 1
        c[1] += end - start
        if key.startswith("k_pick_final"):
            picks += 1
            st = 1 if picks < k else 2
        if key.startswith("k_commit"):
            st = None
    print(f"{rounds} rounds")
    for title, tab in zip(stages, per):
        tot = sum(v[1] for v in tab.values())
        print(f"{title}: {tot / 1e6 / max(1, rounds):.3f} ms/round")
        for key, (n, ns) in sorted(tab.items(), key=lambda x: -x[1][1])[:8]:
            print(f"  {key[:40]:40s} {n / max(1, rounds):7.2f}/round  {ns / 1e6 / max(1, rounds):8.3f} ms/round"
                  f"  avg {ns / n / 1e3:9.2f} us")


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


def phase_table(trace, wl, path):
    """Per-phase times of one profiled round of the persistent path, from SD2_DBG_TRACE (device clock
    at 100 MHz as seen by workgroup 0: entry 0 the start of launch j, entry p + 1 the end of its
    phase p).  Phases of a launch: per layer Q|K|V (+ RoPE, cache append; layer 0 also stages the
    embedding), attention, O, gate|up, down, then the LM head.  Writes a markdown table."""
    import numpy as np
    kinds = ["qkv", "attn", "o", "gu", "down"]
    lines = ["| launch | total us | " + " | ".join(f"{k} us (median per layer)" for k in kinds) + " | LM head us |",
             "|---|---|" + "---|" * len(kinds) + "---|"]
    for j in range(0, wl.k + 1):
        L = wl.verifier.n_layers if j == 0 else wl.drafter.n_layers
        n = 5 * L + 1
        t = trace[j, : n + 1].astype(np.float64) / 100.0
        if not (t[1:] >= t[:-1]).all() or t[-1] <= t[0]:
            continue
        d = np.diff(t)
        per = [np.median(d[i : 5 * L : 5]) for i in range(5)]
        name = "verify pass (k_mk<128>)" if j == 0 else f"drafter step {j} (k_mk<64>)"
        lines.append(f"| {name} | {t[-1] - t[0]:.1f} | " + " | ".join(f"{v:.2f}" for v in per) + f" | {d[-1]:.2f} |")
    txt = "\n".join(lines) + "\n"
    log("phase trace:\n" + txt)
    if path:
        with open(path, "w") as f:
            f.write(txt)


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def discover(eng, t_tok, t_len, wl):
    """One generation with the host reading the state after every round: the number of rounds a
    generation takes and every round's start length and active flag per sequence.  A generation
    is deterministic (fixed Philox stream, fixed reduction orders), so later generations replay
    exactly these rounds without host synchronisation."""
    import torch

    eng.prefill(t_tok, t_len, wl.max_prompt)
    rounds = []
    while True:
        st = eng.state()
        if all(s["done"] for s in st[: wl.batch]):
            break
        rounds.append([(s["t"], not s["done"]) for s in st[: wl.batch]])
        eng.round()
        torch.cuda.synchronize()
        if len(rounds) > wl.new_tokens + 8:
            raise RuntimeError("generation did not finish within new_tokens rounds")
    st = eng.state()
    produced = sum(s["produced"] for s in st[: wl.batch])
    return rounds, produced


def generation(eng, t_tok, t_len, wl, nrounds, stream, evs=None):
    """Prefill + nrounds rounds, enqueued without host synchronisation; with `evs` (nrounds + 2
    events) an event is recorded before the prefill, after it and after every round."""
    if evs is not None:
        evs[0].record(stream)
    eng.prefill(t_tok, t_len, wl.max_prompt)
    if evs is not None:
        evs[1].record(stream)
    for r in range(nrounds):
        eng.round()
        if evs is not None:
            evs[r + 2].record(stream)


def gen_bytes(wl, rounds, steering):
    """Algorithmic bytes of every round of a generation (active sequences at their start lengths)."""
    out = []
    for rnd in rounds:
        w_b, kv = 0.0, 0.0
        for t, active in rnd:
            if not active:
                continue
            w, kvv, kvd = round_bytes(wl, t, steering)
            w_b = w
            kv += kvv + kvd
        out.append((w_b, kv))
    return out


def timed_generations(eng, t_tok, t_len, wl, nrounds, steps, stream):
    """K generations between two synchronisations; returns total ms, per-generation prefill ms
    and every round's ms."""
    import torch

    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(nrounds + 2)] for _ in range(steps)]
    torch.cuda.synchronize()
    t_start = time.time()
    for g in range(steps):
        generation(eng, t_tok, t_len, wl, nrounds, stream, evs[g])
    torch.cuda.synchronize()
    wall = time.time() - t_start
    total = evs[0][0].elapsed_time(evs[-1][-1])
    prefill = [e[0].elapsed_time(e[1]) for e in evs]
    rounds = [e[r + 1].elapsed_time(e[r + 2]) for e in evs for r in range(nrounds)]
    return total, wall, prefill, rounds


def main():
    import sd2_inputs as si

    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20, help="timed generations (prefill + every round to new_tokens)")
    ap.add_argument("--warmup", type=int, default=3, help="untimed generations before them")
    ap.add_argument("--workload", default=si.LLAMA8B.name, choices=list(si.BY_NAME))
    ap.add_argument("--prof-generations", type=int, default=1,
                    help="generations replayed with a HIP event pair around every launch (kernel roofline)")
    ap.add_argument("--cpu-budget", type=float, default=20.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-steer-overhead", action="store_true",
                    help="skip the unsteered-drafter generations that give steer_overhead_ms")
    ap.add_argument("--steering", choices=["input", "mlp", "mlp-out"], default="input",
                    help="input: s = W_s h added to the drafter's input embeddings; mlp: the paper's eq. (2) "
                         "per-layer up-projection biases from three verifier layers; mlp-out: its ablation "
                         "with one bias after every drafter MLP (no CPU baseline for either)")
    ap.add_argument("--calib-copy", action="store_true",
                    help="after the rounds, copy one 1 GiB buffer (a plain copy of known size, the reference "
                         "point for scaling hardware traffic counters)")
    ap.add_argument("--phase-trace", metavar="PATH",
                    help="after the timed generations, profile one round of the persistent path and write its "
                         "per-phase times (SD2_DBG_TRACE) as a markdown table to PATH")
    ap.add_argument("--maps-out", metavar="PATH",
                    help="write this process's /proc/self/maps to PATH after teardown (resolves the frames "
                         "of a crash at exit)")
    ap.add_argument("--summarize-trace", metavar="KERNEL_TRACE_CSV",
                    help="print the per-round breakdown of a rocprofv3 kernel trace of this script and exit")
    ap.add_argument("--summarize-stages", metavar="KERNEL_TRACE_CSV",
                    help="print the per-stage breakdown (drafter steps, verify pass) of the rounds of a "
                         "rocprofv3 kernel trace of this script with --workload, and exit")
    ap.add_argument("--summarize-pmc", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="print k_mk HBM traffic from two rocprofv3 --pmc runs of this script with "
                         "--calib-copy and exit")
    ap.add_argument("--write-traffic", action="store_true", help="with --summarize-pmc: store the result")
    args = ap.parse_args()
    if args.summarize_trace:
        summarize_trace(args.summarize_trace)
        return
    if args.summarize_pmc:
        summarize_pmc(*args.summarize_pmc, TRAFFIC_FILE if args.write_traffic else None)
        return
    if args.summarize_stages:
        summarize_stages(args.summarize_stages, si.BY_NAME[args.workload].k)
        return
    if args.gpus != 1:
        print(f"bench.py measures one GPU only (the round runs on one device); --gpus {args.gpus} is not supported", file=sys.stderr)
        sys.exit(2)
    if args.steps < 1:
        print("--steps must be at least 1", file=sys.stderr)
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
    engines = []
    with torch.cuda.stream(stream):
        steer_form = {"input": B.STEER_INPUT, "mlp": B.STEER_MLP, "mlp-out": B.STEER_MLP_OUT}[args.steering]
        eng = B.Engine(B.config_of(wl, steering=steer_form), models[0], models[1], ws_dev, stream=stream,
                       device=dev, mlp=mlp_dev)
        engines.append(eng)
        t_tok = torch.from_numpy(toks).to(dev)
        t_len = torch.from_numpy(lens).to(dev)
        torch.cuda.synchronize()
        # warm-up: the first generation (host reads the state after every round) finds the rounds
        tw = time.time()
        rounds, produced = discover(eng, t_tok, t_len, wl)
        nr = len(rounds)
        log(f"generation: {nr} rounds, {produced} tokens ({time.time() - tw:.2f}s with host reads)")
        for _ in range(max(0, args.warmup - 1)):
            generation(eng, t_tok, t_len, wl, nr, stream)
        torch.cuda.synchronize()
        total_ms, wall_s, prefill_ms, round_ms = timed_generations(eng, t_tok, t_len, wl, nr, args.steps, stream)
        st_end = eng.state()
        assert all(s["done"] for s in st_end[: wl.batch]), "a timed generation did not finish"
        assert sum(s["produced"] for s in st_end[: wl.batch]) == produced, "generations differ"
        log(f"timed {args.steps} generations: {total_ms:.1f} ms (host clock {wall_s * 1e3:.1f} ms)")
        # kernel-level timing: HIP events around every launch of whole replayed generations
        prof = {c: [0, 0.0, 0.0] for c in (B.PROF_PROGRAM, B.PROF_GEMV, B.PROF_ATTN, B.PROF_SAMPLER, B.PROF_OTHER)}
        kv_prof = 0.0
        gb = gen_bytes(wl, rounds, args.steering)
        for _ in range(args.prof_generations):
            eng.prefill(t_tok, t_len, wl.max_prompt)
            eng.profile(True)
            for r in range(nr):
                eng.round()
                for c in prof:
                    n, pms, pby = eng.profile_read(c)
                    prof[c][0] += n
                    prof[c][1] += pms
                    prof[c][2] += pby
                kv_prof += gb[r][1]
            eng.profile(False)
        torch.cuda.synchronize()
        if args.phase_trace and int(eng.debug(B.DBG_PATH)[0]) == 1:
            # one round of a fresh generation at its prompt's length, every phase timed on device
            eng.prefill(t_tok, t_len, wl.max_prompt)
            eng.profile(True)
            eng.round()
            eng.profile(False)
            torch.cuda.synchronize()
            phase_table(eng.debug(B.DBG_TRACE), wl, args.phase_trace)
        # steering overhead: the same generation with the unsteered (pretrained) drafter
        overhead = None
        if not args.no_steer_overhead:
            e0 = B.Engine(B.config_of(wl, steering=B.STEER_NONE), models[0], models[1], None, stream=stream,
                          device=dev)
            engines.append(e0)
            r0, _ = discover(e0, t_tok, t_len, wl)
            gens0 = max(1, min(args.steps, 5))
            _, _, _, rms0 = timed_generations(e0, t_tok, t_len, wl, len(r0), gens0, stream)
            steered = sum(round_ms) / len(round_ms)
            unsteered = sum(rms0) / len(rms0)
            overhead = {"steer_overhead_ms": steered - unsteered, "round_ms_steered_mean": steered,
                        "round_ms_unsteered_mean": unsteered, "unsteered_generations": gens0,
                        "unsteered_rounds_per_generation": len(r0)}
            log(f"steering overhead: {steered:.3f} vs {unsteered:.3f} ms per round (unsteered drafter)")
        if args.calib_copy:
            src = torch.empty(1 << 30, dtype=torch.uint8, device=dev).fill_(1)
            dst = torch.empty_like(src)
            torch.cuda.synchronize()
            dst.copy_(src)
            torch.cuda.synchronize()
            del src, dst

    tokens = produced * args.steps
    sec = total_ms / 1e3
    rsec = sum(round_ms) / 1e3
    sorted_r = sorted(round_ms)
    w_tot = sum(w for w, _ in gb) * args.steps
    kv_tot = sum(kv for _, kv in gb) * args.steps
    bytes_round = (w_tot + kv_tot) / (nr * args.steps)
    ms_round = sum(round_ms) / len(round_ms)
    hbm_frac = (w_tot + kv_tot) / rsec / 1e9 / PEAK_HBM_GBS
    tau = produced / max(1, sum(sum(a for _, a in rnd) for rnd in rounds))
    # roofline of the dominant kernel: the persistent launches (weights they stream, from the
    # library, plus the KV rows their attention phases read, from the sequence lengths)
    p_n, p_ms, p_by = prof[B.PROF_PROGRAM]
    if p_n:
        r_kernel = ("k_mk (persistent launch: one per drafter step, one per verify pass; every projection, "
                    "attention and LM head of that forward)")
        g_n, g_ms, g_by = p_n, p_ms, p_by + kv_prof
    else:
        r_kernel = "k_wsgemv (every weight-streaming projection: QKV, O, gate|up, down, LM heads, W_s)"
        g_n, g_ms, g_by = prof[B.PROF_GEMV]
    gemv_gbs = g_by / (g_ms / 1e3) / 1e9 if g_ms > 0 else 0.0
    npr = max(1, args.prof_generations * nr)
    log(f"round: {ms_round:.3f} ms mean, {bytes_round / 1e9:.3f} GB algorithmic -> {hbm_frac:.1%} of HBM")
    for c, name in ((B.PROF_PROGRAM, "program"), (B.PROF_GEMV, "gemv"), (B.PROF_ATTN, "attn"),
                    (B.PROF_SAMPLER, "sampler"), (B.PROF_OTHER, "other")):
        n, pms, pby = prof[c]
        log(f"  {name}: {n / npr:.0f} launches/round, {pms / npr:.3f} ms/round"
            + (f", {pby / (pms / 1e3) / 1e9:.0f} GB/s" if pby and pms else ""))

    result = {
        "metric": "generated tokens/s at 1 GPU (one step = one whole generation: prefill + every SD2 round "
                  "to new_tokens)",
        "value": tokens / sec,
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": total_ms / args.steps,
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
        "tokens_per_generation": produced,
        "rounds_per_generation": nr,
        "decode_tokens_per_s": tokens / rsec,
        "round_ms_mean": ms_round,
        "round_ms_p50": sorted_r[len(sorted_r) // 2],
        "round_ms_p90": sorted_r[min(len(sorted_r) - 1, (9 * len(sorted_r)) // 10)],
        "prefill_ms_mean": sum(prefill_ms) / len(prefill_ms),
        "block_efficiency": tau,
        "round_bytes_mean": bytes_round,
        "round_hbm_frac": hbm_frac,
        "roofline": {"bound": "hbm", "kernel": r_kernel,
                     "achieved": gemv_gbs, "peak": PEAK_HBM_GBS, "unit": "GB/s", "frac": gemv_gbs / PEAK_HBM_GBS,
                     "traffic": stored_traffic(wl.name) if p_n and args.steering == "input" else None,
                     "launches_per_round": g_n / npr,
                     "avg_launch_us": g_ms / max(1, g_n) * 1e3,
                     "bytes_per_launch": g_by / max(1, g_n)},
        "cpu_baseline": None,
    }
    if overhead:
        result.update(overhead)
    if not args.no_cpu_baseline and args.steering == "input":
        result["cpu_baseline"] = cpu_baseline(wl, host[0], host[1], ws, toks, lens, args.cpu_budget)
    # teardown in order before the interpreter exits: handles, then device tensors, then torch's cache
    torch.cuda.synchronize()
    for e in engines:
        e.close()
    del eng, engines, models, ws_dev, mlp_dev, t_tok, t_len
    torch.cuda.synchronize()
    torch.cuda.empty_cache()
    print(json.dumps(result), flush=True)
    if args.maps_out:
        with open("/proc/self/maps") as f, open(args.maps_out, "w") as g:
            g.write(f.read())


if __name__ == "__main__":
    main()
