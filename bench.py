"""Throughput of the MI355X LightBeam decoding path on one GPU.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload c4] [--fusion-scorer lm] [--merge max]

One step decodes one whole batch of the workload (LB_BEGIN | LB_END over all
frames; streaming workloads are fed chunk by chunk) with the inputs already in
HBM.  Prints ONE JSON line: beam-token expansions per second (value), decoded
audio-seconds per wall-second, per-stream real-time factor, the HBM roofline of
the dominant kernel (per-launch durations from HIP events recorded on the
decode stream) and the CPU oracle timed on a bounded sample of the workload.
With --fusion-scorer lm the fusion scores travel the external round trip
(lb_fusion_request / lb_fusion_scores) from a small random causal word LM, and
the line adds the round trip's breakdown (no CPU baseline in that mode).
"""

from __future__ import annotations

import argparse
import json
import os
import sys
import threading
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "beam-token expansions/sec and decoded audio-sec per wall-sec (RTF) on 1 MI355X"
HBM_PEAK_GBS = 8000.0
LINE_BYTES = 64          # one hash-table bucket = one 64-B line


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", default="c4")
    ap.add_argument("--cpu-sample", type=int, default=0,
                    help="utterances decoded by the CPU oracle (0 = four per host thread, at most 16 threads)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-profile", action="store_true", help="skip per-kernel event timing")
    ap.add_argument("--merge", choices=("lse", "max"), default="lse",
                    help="max: paths into one prefix recombined by their maximum (the best alignment, App. E.1) "
                         "instead of log-sum-exp; the committed traffic and parity figures are for log-sum-exp, "
                         "so the line reports them as null")
    ap.add_argument("--fusion-scorer", choices=("synthetic", "lm"), default="synthetic",
                    help="lm: fusion scores come back through the external round trip from a small "
                         "randomly initialised causal word LM (the LLM stand-in)")
    ap.add_argument("--gather-ceiling", type=float, default=0.0, metavar="GB",
                    help="only time random 64-B line gathers (lb_measure_gather) from a device table of GB "
                         "gigabytes, the access pattern of the n-gram lookups, and exit")
    ap.add_argument("--gather-lines", type=int, default=4_500_000,
                    help="lines gathered per pass in --gather-ceiling (default: about one c4 decode's lookups)")
    ap.add_argument("--copy-calibration", type=int, default=0, metavar="MIB",
                    help="only run a plain device copy of MIB MiB (reads and writes MIB MiB) and exit; "
                         "its FETCH_SIZE / WRITE_SIZE counters calibrate the HBM traffic figures")
    return ap.parse_args()


def copy_calibration(mib: int) -> None:
    import torch
    n = mib * (1 << 20) // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda:0")
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    for _ in range(3):
        torch.mul(src, 1.0, out=dst)
    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    ev0.record()
    torch.mul(src, 1.0, out=dst)
    ev1.record()
    torch.cuda.synchronize()
    ms = ev0.elapsed_time(ev1)
    print(json.dumps({"copy_calibration_mib": mib, "bytes_read": n * 4, "bytes_written": n * 4,
                      "ms": ms, "GBps_read_plus_write": 2 * n * 4 / (ms * 1e-3) / 1e9}), flush=True)


def gather_bandwidth(gb: float, lines: int, reps: int = 5) -> dict:
    """Random 64-B line gathers (lb_measure_gather) from a device table of `gb`
    GB: the n-gram probes' access pattern (one line per probe, uniformly random
    over the tables).  Best of `reps` passes, timed with events on the stream
    of the gathers."""
    import torch
    import paper_2603_14002_amd as lbm
    n_lines = max(1, int(gb * 1e9) // 64)
    table = torch.empty(n_lines * 16, dtype=torch.float32, device="cuda:0")
    threads = (lines + 7) // 8
    out = torch.empty(threads, dtype=torch.int32, device="cuda:0")
    stream = torch.cuda.current_stream()
    lbm.lb_measure_gather(table, n_lines, lines, 260314002, out, threads, stream)
    best = float("inf")
    for r in range(reps):
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        lbm.lb_measure_gather(table, n_lines, lines, 260314002 + r + 1, out, threads, stream)
        e1.record(stream)
        torch.cuda.synchronize()
        best = min(best, e0.elapsed_time(e1))
    del table, out
    torch.cuda.empty_cache()
    return {"table_GB": n_lines * 64 / 1e9, "lines": lines, "ms": best,
            "GBps": lines * 64.0 / (best * 1e-3) / 1e9, "kernel": "k_gather_probe (lb_measure_gather)"}


def gather_ceiling(gb: float, lines: int) -> None:
    print(json.dumps(gather_bandwidth(gb, lines)), flush=True)


def kernel_source_hash() -> str:
    """The library's build id for the sources in this tree (sha256 over the
    sources without comments and spacing, and the build flags); a committed
    traffic or parity figure is valid only for the code it was measured on."""
    from paper_2603_14002_amd.build import source_hash
    return source_hash()


def measured_traffic(workload: str):
    """HBM bytes per k_decode launch from the committed rocprofv3 summary
    (FETCH_SIZE and WRITE_SIZE, each scaled by what the counter reads for a
    plain copy), or None when there is none for this workload or the kernel
    sources changed since it was taken."""
    path = os.path.join(ROOT, "profiles", f"k_decode_{workload}.md")
    if not os.path.exists(path):
        return None
    vals = {}
    with open(path) as fh:
        for line in fh:
            if line.startswith("- ") and ": " in line:
                k, v = line[2:].split(": ", 1)
                vals[k.strip("` ")] = v.strip().strip("`")
    if vals.get("kernel_source_sha256") != kernel_source_hash():
        return None
    try:
        return float(vals["traffic_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def algorithmic_bytes(s, B, T, p, lp):
    """Bytes the method itself moves in the counted work (all launches of the
    pass), per unit of work: a 164-B logit row per stream-frame, a 16-B trie
    node per 41 expansions, the beam state read and written once per call
    (it stays in LDS between frames), a 64-B line per probed hash-table bucket
    (n-gram tables and continuation index) and per lookup the 64-B line of the
    word's unigram entry (the queries of a stream-frame that share context
    and word are looked up once; homophones that back off to their unigram are
    not looked up), an 8-B history-node reference per completed word and
    sub-beam, 8 B per fused sub-beam, and, when the decode launch also writes
    the call's output (no separate output launch), the output rows: B x K x
    (W word ids + a score), 4 B each."""
    state = 48 + 12 * p.subbeams          # key, pkey, a_b, a_nb, total, node, meta + o x (L, hist)
    calls = max(1, int(s.launches[0]))
    parts = {
        "logits": float(s.frames) * 164.0,
        "trie": float(s.expansions) * 16.0 / 41.0,
        "state": 2.0 * calls * B * p.beam * state,
        "ngram_lines": float(s.probe_lines) * LINE_BYTES,
        "unigram_lines": float(s.lm_lookups) * LINE_BYTES,
        "history_nodes": float(s.word_events) * p.subbeams * 8.0,
        "fusion": float(s.fused) * p.subbeams * 8.0,
    }
    import paper_2603_14002_amd as lbm
    if int(s.launches[lbm.KIND_OUTPUT]) == 0:
        parts["output"] = float(calls) * B * p.beam * (lp.max_words_out + 1) * 4.0
    parts["total"] = sum(parts.values())
    return parts


def copy_bandwidth(mib: int = 1024, reps: int = 5) -> float:
    """GB/s (bytes read + written) of a plain device copy of `mib` MiB, best of `reps`."""
    import torch
    n = mib * (1 << 20) // 4
    src = torch.ones(n, dtype=torch.float32, device="cuda:0")
    dst = torch.empty_like(src)
    dst.copy_(src)
    best = float("inf")
    for _ in range(reps):
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record()
        dst.copy_(src)
        e1.record()
        torch.cuda.synchronize()
        best = min(best, e0.elapsed_time(e1))
    del src, dst
    torch.cuda.empty_cache()
    return 2.0 * n * 4 / (best * 1e-3) / 1e9


def committed_parity(workload: str):
    """Parity counts of the full-batch GPU tests for this workload from the
    committed summary, while the library sources hash to the ones they were
    measured on (else None)."""
    path = os.path.join(ROOT, "profiles", f"parity_{workload}.md")
    if not os.path.exists(path):
        return None
    out, sha = {}, None
    with open(path) as fh:
        for line in fh:
            if line.startswith("- kernel_source_sha256: "):
                sha = line.split(": ", 1)[1].strip().strip("`")
            if line.startswith("{") and '"mode"' in line:
                r = json.loads(line)
                out[r["mode"]] = {k: r[k] for k in ("utterances", "exact", "near_tie", "near_tie_excused",
                                                    "tie_divergent", "mismatch", "empty", "hyps_compared")}
    if sha != kernel_source_hash() or not out:
        return None
    return out


def cpu_baseline(d, n_utts: int, threads: int, merge_max: bool = False):
    """The oracle, as it stands, on the first n_utts utterances (full length), one
    utterance per host thread; returns expansions/s and the sample description,
    and the first utterance decoded alone on one core."""
    import oracle
    t0 = time.time()
    orc = oracle.Oracle(d.lexicon, d.lm)
    log(f"oracle loaded in {time.time() - t0:.1f}s")
    op = oracle.params_from(d.workload.params, fusion_seed=d.fusion_seed, merge_max=1 if merge_max else 0)
    L0 = int(d.lengths[0])
    t0 = time.time()
    r0 = orc.decode(d.logits[0, :L0], op, max_hyps=d.workload.params.beam)
    one = time.time() - t0
    single = dict(seconds_per_utterance=one, expansions_per_s=r0.stats["expansions"] / one,
                  rtf=one / (L0 * 0.08), sample=f"utterance 0 ({L0} frames) alone on one thread")
    exps = [0] * n_utts
    frames = [0] * n_utts
    nxt = [0]
    lock = threading.Lock()

    def worker():
        while True:
            with lock:
                b = nxt[0]
                nxt[0] += 1
            if b >= n_utts:
                return
            L = int(d.lengths[b])
            r = orc.decode(d.logits[b, :L], op, max_hyps=d.workload.params.beam)
            exps[b] = r.stats["expansions"]
            frames[b] = L

    t0 = time.time()
    ths = [threading.Thread(target=worker) for _ in range(threads)]
    for t in ths:
        t.start()
    for t in ths:
        t.join()
    wall = time.time() - t0
    orc.close()
    return dict(value=sum(exps) / wall, unit="beam-token expansions/s", cores=threads, kind="oracle",
                sample=f"first {n_utts} utterances of {d.workload.name} (all frames), "
                       f"one per thread on {threads} threads, {wall:.1f}s wall",
                host_cpu_count=os.cpu_count(), audio_sec_per_wall_sec=sum(frames) * 0.08 / wall,
                single_core=single)


def main():
    args = parse()
    if args.copy_calibration:
        copy_calibration(args.copy_calibration)
        return
    if args.gather_ceiling:
        gather_ceiling(args.gather_ceiling, args.gather_lines)
        return
    if args.gpus != 1:
        print(json.dumps({"error": "this decoder runs on one GPU; --gpus N>1 is not supported "
                                   "(streams shard across GPUs with no exchange, see the design notes)"}))
        sys.exit(2)
    import torch

    import paper_2603_14002_amd as lbm
    from workloads import FRAME_SECONDS, load_workload

    t0 = time.time()
    d = load_workload(args.workload)
    wl = d.workload
    p = wl.params
    B, T = d.logits.shape[:2]
    log(f"workload {wl.name}: B={B} T={T} K={p.beam} lm={d.lm.counts} ({time.time() - t0:.1f}s)")
    t0 = time.time()
    external = args.fusion_scorer == "lm"
    if external and p.fusion_interval <= 0:
        raise SystemExit(f"workload {wl.name} has no fusion")
    lp = lbm.make_params(p, max_batch=B, max_frames=T, fusion_seed=d.fusion_seed,
                         fusion_source=lbm.LB_FUSION_EXTERNAL if external else None,
                         merge=lbm.LB_MERGE_MAX if args.merge == "max" else lbm.LB_MERGE_LOGSUMEXP)
    dec = lbm.Decoder(d.lexicon, d.lm, lp)
    log(f"lb_create {time.time() - t0:.1f}s")
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream()
    logits = torch.from_numpy(d.logits).to(dev)
    lengths_np = d.lengths.astype(np.int32)
    K, W = lp.beam, lp.max_words_out
    hyps = torch.empty((B, K, W), dtype=torch.int32, device=dev)
    scores = torch.empty((B, K), dtype=torch.float32, device=dev)
    chunk = wl.chunk
    if chunk > 0:
        nch = (T + chunk - 1) // chunk
        chunks = []
        for c in range(nch):
            lo, hi = c * chunk, min(T, (c + 1) * chunk)
            ln = np.clip(lengths_np - lo, 0, hi - lo).astype(np.int32)
            fl = (lbm.LB_BEGIN if c == 0 else 0) | (lbm.LB_END if c == nch - 1 else 0)
            chunks.append((logits[:, lo:hi].contiguous(), torch.from_numpy(ln).to(dev), hi - lo, fl))
    else:
        chunks = [(logits, torch.from_numpy(lengths_np).to(dev), T, lbm.LB_BEGIN | lbm.LB_END)]

    rt = None
    if external:
        from workloads.fusion_lm import CausalWordLM, RoundTripStats, decode_external
        flm = CausalWordLM(d.lm.vocab_size, d.lm.bos, seed=d.fusion_seed & 0xFFFFFFFF).to(dev)
        fwords = torch.empty((B, K, lp.subbeams, W), dtype=torch.int32, device=dev)
        fnw = torch.empty((B, K, lp.subbeams), dtype=torch.int32, device=dev)
        rt = RoundTripStats()

    def step():
        for lg, ln, tc, fl in chunks:
            if external:
                decode_external(lbm, dec, lg, ln, fl, flm.score, hyps, scores, fwords, fnw, stream=stream,
                                stats=rt)
                continue
            st = lbm.lb_decode_batch(dec.handle, lg, ln, B, tc, fl, stream, hyps, scores)
            assert st == lbm.LB_OK

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    st = dec.status()
    if st != lbm.LB_OK:
        raise RuntimeError(lbm.lb_last_error())
    def timed_pass(mask):
        """K steps bracketed by HIP events on the decode stream; `mask` selects the
        kernels also timed individually (0: none, so the wall time is clean)."""
        lbm.lb_reset_stats(dec.handle)
        lbm.lb_set_profiling(dec.handle, mask)
        ev0 = torch.cuda.Event(enable_timing=True)
        ev1 = torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        ev0.record(stream)
        for _ in range(args.steps):
            step()
        ev1.record(stream)
        torch.cuda.synchronize()
        lbm.lb_set_profiling(dec.handle, 0)
        return ev0.elapsed_time(ev1), lbm.lb_get_stats(dec.handle)

    # (1) the timed region: no per-kernel events
    if rt is not None:
        rt.__init__()
    wall_ms, s = timed_pass(0)
    rt_clean = None if rt is None else dict(rt.__dict__)
    ms = wall_ms / args.steps
    exp_per_step = s.expansions / args.steps
    audio = float(lengths_np.sum()) * FRAME_SECONDS
    value = exp_per_step / (ms / 1000.0)
    roof = None
    kern = {}
    out_phase, roof_lookup = None, None
    if not args.no_profile:
        # (2) the same K steps with every kernel timed by events carried in its
        # own dispatch: k_decode's duration for the roofline, and the breakdown
        wall_p, sp = timed_pass(lbm.LB_PROFILE_ALL)
        for k, name in enumerate(lbm.KIND_NAMES):
            if sp.timed[k]:
                kern[name] = dict(launches=int(sp.launches[k]), total_ms=sp.kernel_ms[k],
                                  avg_us=1000.0 * sp.kernel_ms[k] / sp.timed[k])
        if kern:
            kern["dominant"] = max(kern, key=lambda k: kern[k]["total_ms"])
        i = lbm.KIND_DECODE
        nl = max(1, int(sp.launches[i]))
        avg_us = 1000.0 * sp.kernel_ms[i] / max(1, sp.timed[i])
        alg = {k: v / nl for k, v in algorithmic_bytes(sp, B, T, p, lp).items()}
        roof = dict(kernel="k_decode", bound="hbm", achieved=alg["total"] / (avg_us * 1e-6) / 1e9,
                    peak=HBM_PEAK_GBS, unit="GB/s", frac=None,
                    traffic=measured_traffic(wl.name) if args.merge == "lse" else None,
                    bytes_per_launch=alg, avg_launch_us=avg_us, launches=nl,
                    timing="start/stop events carried by each k_decode dispatch (hipExtLaunchKernel), "
                           "a second pass of the same steps",
                    wall_ms_per_step_in_that_pass=wall_p / args.steps)
        roof["frac"] = roof["achieved"] / HBM_PEAK_GBS
        roof["copy_GBps"] = copy_bandwidth()
        roof["frac_of_copy"] = roof["achieved"] / roof["copy_GBps"]
        # (3) the same K steps with the decode kernel's phase counters on: each
        # phase's share of the workgroups' cycles, and the n-gram lookup phase
        # against the HBM roofline (its bytes over its share of the launch)
        _, sph = timed_pass(lbm.LB_PROFILE_PHASES)
        cyc = [float(x) for x in sph.phase_cycles]
        tot = sum(cyc)
        if tot > 0:
            share = {n: c / tot for n, c in zip(lbm.PHASE_NAMES, cyc)}
            nl3 = max(1, int(sph.launches[i]))
            look_bytes = ((sph.probe_lines - sph.index_lines) * LINE_BYTES + sph.lm_lookups * LINE_BYTES) / nl3
            look_s = share["ngram_lookup"] * avg_us * 1e-6
            ach = look_bytes / look_s / 1e9 if look_s > 0 else None
            out_phase = dict(share=share, cycles_per_stream_frame={n: c / max(1, sph.frames) for n, c in
                                                                   zip(lbm.PHASE_NAMES, cyc)})
            # the random 64-B gather ceiling over a table as large as the workload's n-gram tables
            lf = lp.lm_load_factor if lp.lm_load_factor > 0 else 0.25
            table_gb = sum(d.lm.counts[1:]) / lf * 16 / 1e9
            ceil = gather_bandwidth(table_gb, max(4_000_000, int(look_bytes // LINE_BYTES)))
            roof_lookup = dict(
                kernel="k_decode n-gram lookup phase", bound="hbm", achieved=ach, peak=HBM_PEAK_GBS, unit="GB/s",
                frac=None if ach is None else ach / HBM_PEAK_GBS,
                frac_of_copy=None if ach is None else ach / roof["copy_GBps"],
                gather_ceiling=ceil,
                frac_of_gather_ceiling=None if ach is None else ach / ceil["GBps"],
                traffic=None, bytes_per_launch=look_bytes,
                lines_per_launch=(sph.probe_lines - sph.index_lines) / nl3,
                lookups_per_launch=sph.lm_lookups / nl3,
                phase_seconds_per_launch=look_s,
                timing="the phase's share of the workgroups' clock cycles (s_memtime at its barriers) x the "
                       "event-timed k_decode launch duration; bytes: a 64-B line per probed bucket of the "
                       "n-gram tables and per lookup the unigram entry's line")
        else:
            out_phase, roof_lookup = None, None
    out = {
        "metric": METRIC,
        "value": value,
        "unit": "beam-token expansions/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": ms,
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f64",
        "data": "synthetic",
        "config": {"workload": wl.name, "batch": B, "frames": T, "beam": p.beam, "subbeams": p.subbeams,
                   "lexicon_words": d.lexicon.n_words, "ngrams": int(sum(d.lm.counts)),
                   "fusion_interval": p.fusion_interval, "fusion_top_f": p.fusion_top_f,
                   "chunk": chunk, "merge": args.merge, "parallelism": "none (1 GPU)"},
        "audio_sec_per_wall_sec": audio / (ms / 1000.0),
        "rtf_per_stream": (ms / 1000.0) / (T * FRAME_SECONDS) if chunk == 0
        else (ms / 1000.0) / len(chunks) / (chunk * FRAME_SECONDS),
        "counters": {"expansions_per_step": exp_per_step, "word_events_per_step": s.word_events / args.steps,
                     "lm_queries_per_step": s.lm_queries / args.steps, "fused_per_step": s.fused / args.steps,
                     "lm_lookups_per_step": s.lm_lookups / args.steps,
                     "probe_lines_per_step": s.probe_lines / args.steps},
        "kernels": kern,
        "roofline": roof,
        "roofline_lookup_phase": roof_lookup,
        "phases": out_phase,
        "parity": committed_parity(wl.name) if args.merge == "lse" else None,
    }
    if external:
        n = args.steps
        out["config"]["fusion_scorer"] = ("external round trip: causal word LM (d=256, 2 layers, 4 heads, "
                                          "random init, fp32), distinct sequences in batches of 256")
        out["round_trip"] = {
            "events_per_step": rt_clean["events"] / n,
            "sequences_requested_per_step": rt_clean["requested"] / n,
            "distinct_scored_per_step": rt_clean["scored"] / n,
            "scorer_batches_per_step": rt_clean["batches"] / n,
            "scorer_gpu_ms_per_step": rt_clean["scorer_ms"] / n,
            "decoder_kernels_ms_per_step": sum(v["total_ms"] for k, v in kern.items() if k != "dominant") / n
            if kern else None,
            "note": "scorer_gpu_ms from events around the caller's scoring (torch stream); kernel time from "
                    "the profiled pass; the rest of ms_per_step is host round trips and syncs",
        }
        args.no_cpu_baseline = True
    if not args.no_cpu_baseline:
        threads = min(os.cpu_count() or 1, 16)
        n = args.cpu_sample or 4 * threads
        out["cpu_baseline"] = cpu_baseline(d, min(n, B), threads, merge_max=args.merge == "max")
    dec.close()
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
