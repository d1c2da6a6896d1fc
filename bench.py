"""Benchmark of the TokenTiming verification hot path on one MI355X.

One step = the whole verification path (alignment, transfer, verification) over one
batch of synthetic input (default: 256 streams, K=8 draft tokens, V_d=128,256,
V_t=151,936, w=8), issued as tt_step (one fused kernel when the batch fits it) or, with
--path calls, as tt_align + tt_transfer + tt_verify.  Inputs are resident in HBM before
timing starts.  The probability rows are replicated (--replicas) and consecutive steps
read different replicas, so the 256 MB Infinity Cache cannot serve a row from the
previous step.

Prints one JSON line: verified draft tokens/s for the step, per-call times, DTW cells/s,
the dominant kernel against its roofline, and the CPU oracle timed on the host cores on
a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import ctypes
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

HBM_PEAK_GBS = 8000.0


def band_cells(K, M, w):
    """In-band cells per pair: |i - j| <= max(w, |K-M|) (w < 0: all K*M)."""
    K = np.asarray(K, np.int64)
    M = np.asarray(M, np.int64)
    L = np.where(w < 0, np.maximum(K, M), np.maximum(w, np.abs(K - M)))
    total = 0
    for k, m, l in zip(K, M, L):
        i = np.arange(1, k + 1)
        total += int(np.maximum(0, np.minimum(m, i + l) - np.maximum(1, i - l) + 1).sum())
    return total


def source_digest(files):
    """sha256 of kernel sources: counter figures taken from another version of the kernel
    are not reported."""
    import hashlib
    h = hashlib.sha256()
    for f in files:
        with open(os.path.join(ROOT, "paper_2510_15545_amd", "csrc", f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


# sources each measured kernel is built from (a change to any of them voids its counters)
KERNEL_SOURCES = {
    "step_fused": ("step.hip", "dtw_rows.h", "dtw_common.h", "verify_core.h"),
    "verify_row": ("verify.hip", "verify_core.h"),
    "dtw_band": ("dtw.hip", "dtw_common.h"),
    "verify_logits_row": ("logits.hip", "verify_core.h"),
    "verify_tli_row": ("tli.hip", "verify_core.h"),
}
# int32 VALU issue peak of MI355X: 256 CUs x 4 SIMDs x 16 lanes x 2.4 GHz (a wave64 instruction
# occupies its SIMD four cycles), in lane-operations per second
VALU_PEAK_TOPS = 256 * 4 * 16 * 2.4e9 / 1e12


def read_counters(path, workload, kernel):
    """key: value lines of a counter summary, or (None, reason) when the file is missing,
    covers another workload or kernel, or was taken from other kernel sources."""
    if not path or not os.path.exists(path):
        return None, "no counter summary"
    kv = {}
    with open(path) as f:
        for line in f:
            if ":" in line and not line.startswith((" ", "#", "|")):
                k, v = line.split(":", 1)
                kv[k.strip()] = v.strip()
    if kv.get("workload") != workload:
        return None, "counters cover workload %r" % kv.get("workload")
    if kv.get("kernel") != kernel:
        return None, "counters cover kernel %r" % kv.get("kernel")
    if kv.get("source_sha256") != source_digest(KERNEL_SOURCES[kernel]):
        return None, "kernel changed since the counters were taken"
    return kv, ""


def copy_calibration(args, dev):
    """With --copy-calib-mb: one plain device-to-device copy of that many MiB after the timed
    calls, whose counter readings scale a kernel's FETCH_SIZE and WRITE_SIZE to bytes."""
    import torch

    if not args.copy_calib_mb:
        return
    src = torch.empty(args.copy_calib_mb * (1 << 20) // 4, dtype=torch.float32, device=dev).fill_(1.0)
    dst = torch.empty_like(src)
    torch.cuda.synchronize()
    dst.copy_(src)
    torch.cuda.synchronize()


def read_traffic(path, workload, kernel):
    """HBM bytes per launch of `kernel` from a counter summary (key: value lines), or None
    when the summary does not apply (see read_counters)."""
    kv, why = read_counters(path, workload, kernel)
    if kv is None:
        return None, why
    return int(kv["traffic_bytes_per_launch"]), "FETCH_SIZE x %s + WRITE_SIZE x %s" % (
        kv.get("fetch_scale"), kv.get("write_scale"))


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=200)
    ap.add_argument("--warmup", type=int, default=20)
    ap.add_argument("--workload", type=int, default=3, help="synthetic workload 1-5")
    ap.add_argument("--streams", type=int, default=None, help="override the stream count")
    ap.add_argument("--w", type=int, default=8)
    ap.add_argument("--replicas", type=int, default=4)
    ap.add_argument("--path", choices=["step", "calls"], default="step",
                    help="step: one tt_step call per step; calls: tt_align + tt_transfer + tt_verify")
    ap.add_argument("--eager", action="store_true", help="launch every call from Python (no HIP graph)")
    ap.add_argument("--graph-steps", type=int, default=8, help="consecutive steps captured in one HIP graph")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-extras", action="store_true",
                    help="leave out the DTW stress batch and the high-acceptance batch of the default run")
    ap.add_argument("--cpu-seconds", type=float, default=12.0)
    ap.add_argument("--copy-calib-mb", type=int, default=0,
                    help="also run one plain device copy of this many MiB (counter calibration)")
    ap.add_argument("--only", choices=["step", "verify", "align", "transfer"], default=None,
                    help="after the timed steps, loop only this call (for profiler passes)")
    ap.add_argument("--dense", action="store_true",
                    help="standard speculative sampling with dense proposals over one vocabulary "
                         "(tt_verify_dense) on 256 streams x M=8 at V=151,936 instead of the TokenTiming path")
    ap.add_argument("--lse", action="store_true",
                    help="with --logits: pass per-row log-sum-exp values (computed on the GPU beforehand)")
    ap.add_argument("--logits", action="store_true",
                    help="verification from bf16 target logits and a temperature (tt_verify_logits) on the "
                         "benchmark's 256 streams at V_t=151,936 instead of fp32 probability rows")
    ap.add_argument("--tli", action="store_true",
                    help="standard speculative sampling with the Token-Level Intersection proposal (App. D "
                         "Alg. 3) on 256 streams x M=8 at the benchmark's vocabularies: tt_verify_tli (q' formed "
                         "on the fly, with and without the drafter's masses) against tt_tli_proposal + "
                         "tt_verify_dense")
    ap.add_argument("--read-ceiling", action="store_true",
                    help="time plain device reads of the benchmark's bytes (256 rows x 151,936 fp32, rotating "
                         "replicas) with a library reduction and a device-to-device copy: the practical HBM "
                         "read rate the verification's rows are compared against")
    ap.add_argument("--phase-stamps", action="store_true",
                    help="with a library built with -DTT_PHASE_STAMPS: where verify_row's and step_fused's time "
                         "goes on the benchmark batch (per-workgroup real-time stamps at the phase boundaries)")
    ap.add_argument("--traffic", type=str, default=None,
                    help="counter summary with the measured HBM bytes per launch of the dominant kernel "
                         "(default: profiles/<kernel>_counters.txt)")
    return ap.parse_args()


def main():
    args = parse()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU: the verification path runs per stream on a single device; "
              "run with --gpus 1", file=sys.stderr)
        sys.exit(2)

    if args.dense:
        return main_dense(args)
    if args.tli:
        return main_tli(args)
    if args.logits:
        return main_logits(args)
    if args.read_ceiling:
        return main_read_ceiling(args)
    if args.phase_stamps:
        return main_phase_stamps(args)

    import torch

    import paper_2510_15545_amd as tt
    from paper_2510_15545_amd import synth

    tt.lib()  # fail loudly if the HIP library is not built
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)

    t_gen = time.time()
    wl0 = synth.make(args.workload, n_streams=args.streams, w=args.w)
    stage = wl0.prob if args.workload == 4 else wl0
    t_gen = time.time() - t_gen

    def t(a):
        return torch.from_numpy(np.ascontiguousarray(a)).to(dev)

    # alignment inputs (the long pairs for workload 4, the stream batch otherwise)
    A = wl0
    mtb = max(A.vocab_d.max_len, A.vocab_t.max_len)
    vd = tt.Vocab.from_host(A.vocab_d.data, A.vocab_d.offsets, A.vocab_d.max_len, dev)
    vt = tt.Vocab.from_host(A.vocab_t.data, A.vocab_t.offsets, A.vocab_t.max_len, dev)
    a_di, a_do, a_ti, a_to = t(A.draft_ids), t(A.draft_off), t(A.target_ids), t(A.target_off)
    a_maxk, a_maxm = max(1, A.max_k), max(1, A.max_m)
    npath = tt.path_capacity(A.draft_off[-1], A.target_off[-1])
    a_ws = tt.align_workspace(A.n, a_maxk, a_maxm, args.w, mtb, dev)
    a_out = tt.align(vd, vt, a_di, a_do, a_ti, a_to, args.w, a_maxk, a_maxm, n_path=npath, workspace=a_ws)

    S = stage
    s_di, s_do, s_ti, s_to = t(S.draft_ids), t(S.draft_off), t(S.target_ids), t(S.target_off)
    s_vi = t(S.verify_ids)
    s_maxk, s_maxm = max(1, S.max_k), max(1, S.max_m)
    s_npath = tt.path_capacity(S.draft_off[-1], S.target_off[-1])
    if args.workload == 4:  # the probability stage aligns its own short streams
        s_out = tt.align(vd, vt, s_di, s_do, s_ti, s_to, args.w, s_maxk, s_maxm, n_path=s_npath)
    else:
        s_out = a_out
    R = max(1, args.replicas)
    draft_probs = t(S.draft_probs)
    target_probs = [t(S.target_probs)]
    for _ in range(R - 1):
        target_probs.append(target_probs[0].clone())
    ua, us = t(S.u_accept), t(S.u_sample)
    q = torch.empty(max(1, int(S.target_off[-1])), dtype=torch.float32, device=dev)
    n = S.n
    nacc = torch.empty(n, dtype=torch.int32, device=dev)
    tok = torch.empty(n, dtype=torch.int32, device=dev)
    ws = tt.verify_workspace(n, S.v_t, dev)
    # tt_step aligns and verifies the same target ids: the long-pair workload's probability
    # stage indexes its rows with other ids, so it keeps the three calls
    step_ok = args.path == "step" and args.workload != 4
    if step_ok:
        st_ws = tt.step_workspace(n, S.v_t, s_maxk, s_maxm, args.w, mtb, dev)
        st_out = (torch.empty(n, dtype=torch.int32, device=dev), torch.empty(n, dtype=torch.int32, device=dev),
                  torch.empty(max(1, s_npath), dtype=torch.int32, device=dev),
                  torch.empty(max(1, int(S.target_off[-1])), dtype=torch.int32, device=dev), q, nacc, tok, None)
    torch.cuda.synchronize()
    del wl0  # keep host memory for the CPU leg only where needed

    def do_align():
        tt.align(vd, vt, a_di, a_do, a_ti, a_to, args.w, a_maxk, a_maxm, out=a_out, workspace=a_ws)

    def do_transfer():
        tt.transfer(S.v_d, s_di, s_do, s_to, s_out[3], draft_probs, out=q)

    def do_verify(r):
        tt.verify(S.v_t, s_vi, s_to, q, target_probs[r], ua, us, s_maxm, workspace=ws, out=(nacc, tok, None))

    def do_step(r):
        tt.step(vd, vt, S.v_d, S.v_t, s_di, s_do, s_ti, s_to, args.w, s_maxk, s_maxm, draft_probs,
                target_probs[r], ua, us, workspace=st_ws, out=st_out)

    def calls(r):
        do_align()
        if args.workload == 4:
            tt.align(vd, vt, s_di, s_do, s_ti, s_to, args.w, s_maxk, s_maxm, out=s_out)
        do_transfer()
        do_verify(r)

    step = do_step if step_ok else calls

    def graph_of(fn, k):
        g = torch.cuda.CUDAGraph()
        cap = torch.cuda.Stream()
        cap.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(cap):
            with torch.cuda.graph(g, stream=cap):
                for i in range(k):
                    fn(i)
        torch.cuda.current_stream().wait_stream(cap)
        g.replay()
        torch.cuda.synchronize()
        return g

    def run_steps(fn, k):
        """ms per step over exactly k steps, step i reading replica i % R.  With graphs, each
        HIP graph holds --graph-steps consecutive steps (one decode step after another, as
        inside a captured serving loop), so the host's graph launch is not charged per step."""
        s0, s1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        if args.eager:
            torch.cuda.synchronize()
            s0.record()
            for i in range(k):
                fn(i % R)
            s1.record()
            torch.cuda.synchronize()
            return s0.elapsed_time(s1) / k
        gs = max(1, min(args.graph_steps, k))
        full = graph_of(lambda i: fn(i % R), gs)  # gs is a multiple of R or covers k
        rest = k % gs
        tail = graph_of(lambda i: fn(i % R), rest) if rest else None
        torch.cuda.synchronize()
        s0.record()
        for _ in range(k // gs):
            full.replay()
        if tail is not None:
            tail.replay()
        s1.record()
        torch.cuda.synchronize()
        return s0.elapsed_time(s1) / k

    for i in range(args.warmup):
        step(i % R)
        if step_ok:
            calls(i % R)
    torch.cuda.synchronize()

    ms_step = run_steps(step, args.steps)
    ms_calls = run_steps(calls, args.steps) if step_ok else ms_step
    step_outputs = None
    if step_ok:  # the fused path's results must equal the three calls' on this input
        do_step(0)
        torch.cuda.synchronize()
        step_outputs = (nacc.clone(), tok.clone(), st_out[0].clone())
        calls(0)
        torch.cuda.synchronize()
        if not (torch.equal(step_outputs[0], nacc) and torch.equal(step_outputs[1], tok) and
                torch.equal(step_outputs[2], s_out[0])):
            print("tt_step and the three calls disagree", file=sys.stderr)
            sys.exit(3)

    # per-call averages: each call alone, 20 back to back inside one HIP graph (rotating
    # replicas), replayed; HIP events on the stream the graph runs on
    def kernel_ms(fn, k=20, reps=10):
        if args.eager:
            s0, s1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            torch.cuda.synchronize()
            s0.record()
            for i in range(k * reps):
                fn(i)
            s1.record()
            torch.cuda.synchronize()
            return s0.elapsed_time(s1) / (k * reps)
        g = graph_of(fn, k)
        s0, s1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        s0.record()
        for _ in range(reps):
            g.replay()
        s1.record()
        torch.cuda.synchronize()
        return s0.elapsed_time(s1) / (k * reps)

    times = {"align": kernel_ms(lambda i: do_align()), "transfer": kernel_ms(lambda i: do_transfer()),
             "verify": kernel_ms(lambda i: do_verify(i % R))}
    if step_ok:
        times["step"] = kernel_ms(lambda i: do_step(i % R))
    # the step before alignment (Sec. 4.2.1): draft ids -> proxy target ids by greedy longest
    # match, on the alignment batch; the token index is built once, outside the timing
    vt_index = tt.token_index(vt)
    rt_bytes = int((np.diff(A.vocab_d.offsets)[A.draft_ids]).sum())
    rt_maxb = int(max(np.add.reduceat(np.diff(A.vocab_d.offsets)[A.draft_ids], A.draft_off[:-1])))
    rt_out = (torch.empty(A.n * a_maxm, dtype=torch.int32, device=dev), torch.empty(A.n + 1, dtype=torch.int32, device=dev))
    if rt_maxb <= 4096:  # the per-stream string bound tt_retokenize accepts
        tt.retokenize(vd, vt, vt_index, a_di, a_do, rt_maxb, a_maxm, out=rt_out)
        torch.cuda.synchronize()
        if not (np.array_equal(rt_out[1].cpu().numpy(), A.target_off) and
                np.array_equal(rt_out[0].cpu().numpy()[:int(A.target_off[-1])], A.target_ids)):
            print("tt_retokenize disagrees with the workload's target ids", file=sys.stderr)
            sys.exit(3)
        times["retokenize"] = kernel_ms(
            lambda i: tt.retokenize(vd, vt, vt_index, a_di, a_do, rt_maxb, a_maxm, out=rt_out))
    # side output for choosing w (Fig. CDF, App. K): deviation histogram of the aligned batch
    hist = torch.empty(256, dtype=torch.int32, device=dev)
    times["delta_histogram"] = kernel_ms(
        lambda i: tt.delta_histogram(a_do, a_to, a_out[1], a_out[2], 256, out=hist))
    # Token-Level Intersection proposal (App. D Alg. 3): q' over V_t for every draft row of the
    # batch (one per drafted position); the intersection of the two vocabularies is built once
    tli = None
    if draft_probs.shape[1] == vd.n_tokens:
        d2t, t2d = tt.vocab_intersection(vd, tt.token_index(vd), vt, vt_index)
        tli_out = torch.empty((draft_probs.shape[0], vt.n_tokens), dtype=torch.float32, device=dev)
        times["tli_proposal"] = kernel_ms(lambda i: tt.tli_proposal(d2t, t2d, draft_probs, out=tli_out), reps=3)
        tli_bytes = 4 * draft_probs.shape[0] * (vd.n_tokens + vt.n_tokens)
        tli = {"us": round(times["tli_proposal"] * 1e3, 1), "rows": int(draft_probs.shape[0]),
               "intersection_tokens": int((d2t >= 0).sum().item()),
               "GBps": round(tli_bytes / (times["tli_proposal"] * 1e-3) / 1e9, 1)}
        del tli_out
    if args.only:
        fn = {"step": lambda i: do_step(i % R), "verify": lambda i: do_verify(i % R),
              "align": lambda i: do_align(), "transfer": lambda i: do_transfer()}[args.only]
        kernel_ms(fn, 200)

    copy_calibration(args, dev)

    # ---- derived metrics
    Ka = np.diff(A.draft_off)
    Ma = np.diff(A.target_off)
    cells = band_cells(Ka, Ma, args.w)
    Ks = np.diff(S.draft_off)
    m_s = np.diff(S.target_off)
    verify_bytes = int(n * 4 * S.v_t + 16 * int(m_s.sum()) + 12 * n)
    draft_tokens = int(S.draft_off[-1])
    acc = nacc.cpu().numpy()
    gbs_verify = verify_bytes / (times["verify"] * 1e-3) / 1e9
    cells_per_s = cells / (times["align"] * 1e-3)
    wl_name = synth.SPECS[args.workload].name

    if step_ok and synth_fits_fused(S):
        # algorithmic bytes of one fused launch: the verify stream (one row per stream, t_j,
        # P_t(t_j), u_j per position, u_sample, n_accepted, out_token), the alignment reads
        # (offsets, ids, the tokens' table offsets and bytes, one draft probability per
        # draft token) and its writes (cost, path_len, path, map, q)
        plen = st_out[1].cpu().numpy()
        tok_bytes = (np.diff(A.vocab_d.offsets)[S.draft_ids].sum() + np.diff(A.vocab_t.offsets)[S.target_ids].sum())
        step_bytes = int(n * 4 * S.v_t + 12 * int(m_s.sum()) + 12 * n + 16 * n + 8 * int(Ks.sum() + m_s.sum()) +
                         int(tok_bytes) + 8 * int(Ks.sum()) + 8 * n + 8 * int(plen.sum()) +
                         8 * int(m_s.sum()))
        kname, kbytes, kms = "step_fused", step_bytes, times["step"]
    else:
        kname, kbytes, kms = "verify_row" if n >= 256 else "verify_stream + verify_sample", verify_bytes, \
            times["verify"]
    dominant_calls = max(("align", "transfer", "verify"), key=lambda k: times[k])
    traffic_path = args.traffic or os.path.join(ROOT, "profiles", kname.split()[0] + "_counters.txt")
    traffic, traffic_note = read_traffic(traffic_path, wl_name, kname) if kname in KERNEL_SOURCES else \
        (None, "no counters for this kernel")
    if kname == "step_fused" or dominant_calls == "verify":
        gbs = kbytes / (kms * 1e-3) / 1e9
        roof = {"kernel": kname, "bound": "hbm", "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS, "unit": "GB/s",
                "frac": round(gbs / HBM_PEAK_GBS, 4), "traffic": traffic, "traffic_note": traffic_note,
                "algorithmic_bytes_per_launch": kbytes, "launch_us": round(kms * 1e3, 2)}
    else:
        # the strip alignment kernel is bound by VALU issue: executed VALU lane-operations per
        # second (instruction count from the SQ counter summary) against the VALU peak
        kv, why = read_counters(os.path.join(ROOT, "profiles", "dtw_band_counters.txt"), wl_name, "dtw_band")
        tops = None if kv is None else int(kv["valu_instructions_per_launch"]) * 64 / (times["align"] * 1e-3) / 1e12
        roof = {"kernel": "dtw_band", "bound": "alu",
                "achieved": None if tops is None else round(tops, 3), "peak": round(VALU_PEAK_TOPS, 2),
                "unit": "TOP/s (VALU lane-ops)", "frac": None if tops is None else round(tops / VALU_PEAK_TOPS, 4),
                "traffic": None, "cells_per_s": round(cells_per_s, 1), "launch_us": round(times["align"] * 1e3, 2),
                "counter_note": why or "SQ_INSTS_VALU x 64 lanes per launch",
                "lds_bank_conflict_rate": None if kv is None else float(kv["lds_bank_conflict_rate"])}

    result = {
        "metric": "verified draft tokens/s + DTW cells/s at V_t=151,936; verify HBM GB/s vs peak",
        "value": round(draft_tokens / (ms_step * 1e-3), 1),
        "unit": "draft tokens/s",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms_step, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f32+i64", "data": "synthetic",
        "config": {"workload": wl_name, "streams": n,
                   "draft_tokens_per_step": draft_tokens, "target_positions": int(m_s.sum()),
                   "v_t": S.v_t, "v_d": S.v_d, "w": args.w, "replicas": R,
                   "path": "tt_step" if step_ok else "tt_align+tt_transfer+tt_verify",
                   "launch": "eager" if args.eager else "hip-graph of %d steps" % args.graph_steps},
        "three_call_ms_per_step": round(ms_calls, 5),
        "kernels_ms": {k: round(v, 5) for k, v in times.items()},
        "dtw": {"band_cells": cells, "cells_per_s": round(cells_per_s, 1),
                "full_cells": int((Ka * Ma).sum()),
                "full_cells_per_s": round(int((Ka * Ma).sum()) / (times["align"] * 1e-3), 1),
                "delta_pos_w90": tt.w_at_quantile(hist, 9, 10), "path_cells": int(a_out[1].sum().item())},
        "retokenize": {"us": round(times["retokenize"] * 1e3, 2) if "retokenize" in times else None,
                       "string_bytes": rt_bytes,
                       "target_tokens": int(A.target_off[-1])},
        "throughput": {"target_positions_per_s": round(int(m_s.sum()) / (ms_step * 1e-3), 1),
                       "accepted_drafts_per_s": round(int(acc[acc >= 0].sum()) / (ms_step * 1e-3), 1),
                       "transfer_share_of_three_calls": round(times["transfer"] / (times["align"] + times["transfer"] +
                                                                                   times["verify"]), 4)},
        "tli_proposal": tli,
        "verify": dict({"GBps": round(gbs_verify, 1), "frac_of_peak": round(gbs_verify / HBM_PEAK_GBS, 4),
                        "algorithmic_bytes": verify_bytes}, **acceptance(acc, S.target_off)),
        "roofline": roof,
        "gen_seconds": round(t_gen, 1),
    }
    if args.workload == 3 and args.streams is None and not args.no_extras:
        result["dtw_stress"] = dtw_stress(dev, args.w)
        result["high_acceptance"] = high_acceptance(dev, args, R)

    if not args.no_cpu_baseline:
        nacc_step = step_outputs[0] if step_outputs is not None else nacc
        tok_step = step_outputs[1] if step_outputs is not None else tok
        result["cpu_baseline"] = cpu_baseline(args, S, A, nacc_step, tok_step, s_out, a_out)
    print(json.dumps(result), flush=True)


def main_dense(args):
    """Dense-proposal verification (App. D Alg. 4 over one vocabulary): one step is one
    tt_verify_dense call over the batch; draft and target rows are replicated like the
    TokenTiming path's target rows."""
    import torch

    import paper_2510_15545_amd as tt
    from paper_2510_15545_amd import synth

    tt.lib()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    n_streams = args.streams or 256
    t_gen = time.time()
    D = synth.make_dense(n_streams, 8, 151_936)
    t_gen = time.time() - t_gen

    def t(a):
        return torch.from_numpy(np.ascontiguousarray(a)).to(dev)

    R = max(1, args.replicas)
    ids, off, ua, us = t(D.draft_ids), t(D.off), t(D.u_accept), t(D.u_sample)
    qrows = [t(D.draft_probs)]
    prows = [t(D.target_probs)]
    for _ in range(R - 1):
        qrows.append(qrows[0].clone())
        prows.append(prows[0].clone())
    n = D.n
    nacc = torch.empty(n, dtype=torch.int32, device=dev)
    tok = torch.empty(n, dtype=torch.int32, device=dev)
    ws = tt.verify_workspace(n, D.v, dev)

    def step(r):
        tt.verify_dense(D.v, ids, off, qrows[r], prows[r], ua, us, D.max_m, workspace=ws, out=(nacc, tok, None))

    for i in range(args.warmup):
        step(i % R)
    torch.cuda.synchronize()
    gs = 1 if args.eager else max(1, min(args.graph_steps, args.steps))
    reps = max(1, args.steps // gs)
    s0, s1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    if args.eager:
        s0.record()
        for i in range(reps):
            step(i % R)
        s1.record()
    else:
        g = torch.cuda.CUDAGraph()
        cap = torch.cuda.Stream()
        cap.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(cap):
            with torch.cuda.graph(g, stream=cap):
                for i in range(gs):
                    step(i % R)
        torch.cuda.current_stream().wait_stream(cap)
        g.replay()
        torch.cuda.synchronize()
        s0.record()
        for _ in range(reps):
            g.replay()
        s1.record()
    torch.cuda.synchronize()
    ms = s0.elapsed_time(s1) / (reps * gs)
    step(0)
    torch.cuda.synchronize()
    copy_calibration(args, dev)
    acc = nacc.cpu().numpy()
    m = np.diff(D.off)
    # algorithmic bytes: the target row of every stream, the draft row of every rejected
    # stream, x_j, p_j(x_j), q_j(x_j), u_j per drafted position, u_sample, n_accepted, out_token
    rejected = int((acc < m).sum())
    kbytes = int(n * 4 * D.v + rejected * 4 * D.v + 16 * int(m.sum()) + 12 * n)
    gbs = kbytes / (ms * 1e-3) / 1e9
    wl_name = D.name
    traffic, note = read_traffic(args.traffic or os.path.join(ROOT, "profiles", "verify_row_dense_counters.txt"),
                                 wl_name, "verify_row")
    result = {
        "metric": "verified draft tokens/s, dense proposals (App. D Alg. 4) at V=151,936; verify HBM GB/s vs peak",
        "value": round(int(m.sum()) / (ms * 1e-3), 1), "unit": "draft tokens/s",
        "n_gpus": 1, "steps": reps * gs, "warmup": args.warmup, "ms_per_step": round(ms, 5),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32+i64", "data": "synthetic",
        "config": {"workload": wl_name, "streams": n, "draft_tokens_per_step": int(m.sum()), "v": D.v,
                   "replicas": R, "path": "tt_verify_dense",
                   "launch": "eager" if args.eager else "hip-graph of %d steps" % gs},
        "accept": {"mean_gamma": round(float(acc.mean()), 3), "rejected_streams": rejected},
        "roofline": {"kernel": "verify_row<dense>", "bound": "hbm", "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": round(gbs / HBM_PEAK_GBS, 4), "traffic": traffic, "traffic_note": note,
                     "algorithmic_bytes_per_launch": kbytes, "launch_us": round(ms * 1e3, 2)},
        "gen_seconds": round(t_gen, 1),
    }
    if not args.no_cpu_baseline:
        import oracle

        threads = len(os.sched_getaffinity(0))
        k, t0 = 0, time.time()
        while k == 0 or time.time() - t0 < args.cpu_seconds:
            o_n, o_t, _, _ = oracle.sd_verify(D.v, D.draft_ids, D.off, D.draft_probs, D.target_probs, D.u_accept,
                                              D.u_sample, n_threads=threads)
            k += 1
        dt = (time.time() - t0) / k
        result["cpu_baseline"] = {
            "value": round(int(m.sum()) / dt, 1), "unit": "draft tokens/s", "cores": threads, "kind": "oracle",
            "sample": f"{k} whole steps of the benchmark batch ({n} streams), {dt * 1e3:.1f} ms each",
            "cpu_model": cpu_model(),
            "matches_gpu": bool(np.array_equal(o_n, acc) and np.array_equal(o_t, tok.cpu().numpy()))}
    print(json.dumps(result), flush=True)


def main_phase_stamps(args):
    """Phase times of verify_row and step_fused on the benchmark batch from the stamps a
    -DTT_PHASE_STAMPS build records (the 100 MHz real-time counter at each phase boundary, per
    workgroup, of the last launch): 20 launches back to back in a HIP graph, then the table is
    read; five samples."""
    import torch

    import paper_2510_15545_amd as tt
    from paper_2510_15545_amd import synth

    L = tt.lib()
    if not hasattr(L, "tt_phase_stamps_verify") or not hasattr(L, "tt_phase_stamps_step"):
        print("the library was built without phase stamps: python3 -m paper_2510_15545_amd.build "
              "-DTT_PHASE_STAMPS", file=sys.stderr)
        sys.exit(2)
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    S = synth.make(3, n_streams=args.streams)
    n = S.n

    def t(a):
        return torch.from_numpy(np.ascontiguousarray(a)).to(dev)

    mtb = max(S.vocab_d.max_len, S.vocab_t.max_len)
    vd = tt.Vocab.from_host(S.vocab_d.data, S.vocab_d.offsets, S.vocab_d.max_len, dev)
    vt = tt.Vocab.from_host(S.vocab_t.data, S.vocab_t.offsets, S.vocab_t.max_len, dev)
    di, do, ti, to, vi = t(S.draft_ids), t(S.draft_off), t(S.target_ids), t(S.target_off), t(S.verify_ids)
    mk, mm = max(1, S.max_k), max(1, S.max_m)
    R = max(1, args.replicas)
    dp = t(S.draft_probs)
    tp = [t(S.target_probs)]
    for _ in range(R - 1):
        tp.append(tp[0].clone())
    ua, us = t(S.u_accept), t(S.u_sample)
    a_out = tt.align(vd, vt, di, do, ti, to, args.w, mk, mm)
    q = tt.transfer(S.v_d, di, do, to, a_out[3], dp)
    nacc = torch.empty(n, dtype=torch.int32, device=dev)
    tok = torch.empty(n, dtype=torch.int32, device=dev)
    ws = tt.verify_workspace(n, S.v_t, dev)
    st_ws = tt.step_workspace(n, S.v_t, mk, mm, args.w, mtb, dev)
    st_out = (torch.empty(n, dtype=torch.int32, device=dev), torch.empty(n, dtype=torch.int32, device=dev),
              torch.empty(max(1, tt.path_capacity(S.draft_off[-1], S.target_off[-1])), dtype=torch.int32,
                          device=dev),
              torch.empty(max(1, int(S.target_off[-1])), dtype=torch.int32, device=dev), torch.empty_like(q),
              torch.empty_like(nacc), torch.empty_like(tok), None)
    hip = ctypes.CDLL("libamdhip64.so")
    slots = 16

    def table(unit):
        f = getattr(L, "tt_phase_stamps_" + unit)
        f.restype = ctypes.c_void_p
        buf = np.zeros(n * slots, np.uint64)
        torch.cuda.synchronize()
        if hip.hipMemcpy(buf.ctypes.data_as(ctypes.c_void_p), ctypes.c_void_p(f()), ctypes.c_size_t(buf.nbytes),
                         2) != 0:
            raise RuntimeError("hipMemcpy of the stamp table failed")
        return buf.reshape(n, slots).astype(np.int64)

    def stats(x):
        x = np.asarray(x, np.float64)
        return {"p0": round(float(x.min()), 2), "p50": round(float(np.median(x)), 2),
                "p90": round(float(np.percentile(x, 90)), 2), "p100": round(float(x.max()), 2)}

    kernels = {
        "verify_row": (lambda i: tt.verify(S.v_t, vi, to, q, tp[i % R], ua, us, mm, workspace=ws,
                                           out=(nacc, tok, None)), "verify",
                       [("acceptance scan (wave 0)", 0, 1), ("stream the row (all waves, to the barrier)", 2, 4),
                        ("sample (wave 0)", 4, 5)], 5),
        "step_fused": (lambda i: tt.step(vd, vt, S.v_d, S.v_t, di, do, ti, to, args.w, mk, mm, dp, tp[i % R], ua, us,
                                         workspace=st_ws, out=st_out), "step",
                       [("staging and prefetch", 0, 1), ("distances, recurrence, move tables", 1, 2),
                        ("backtrack, transfer, acceptance", 2, 3), ("stream the row (to the barrier)", 3, 5),
                        ("sample (wave 0)", 5, 6)], 6),
    }
    out = {"metric": "phase times per workgroup (us) on the benchmark batch", "streams": n}
    for name, (fn, unit, phases, last) in kernels.items():
        us_launch = graph_ms(fn, k=20, reps=5) * 1e3
        samples = {ph: [] for ph, _, _ in phases}
        ends, spans, starts = [], [], []
        for _ in range(5):
            graph_ms(fn, k=20, reps=1)
            st = table(unit)
            rel = (st - st[:, 0].min()) / 100.0  # 100 MHz counter -> us
            for ph, a, b in phases:
                samples[ph].extend(rel[:, b] - rel[:, a])
            ends.extend(rel[:, last])
            starts.extend(rel[:, 0])
            spans.append(rel[:, last].max())
        out[name] = {"launch_us_by_events": round(us_launch, 2),
                     "phases": {ph: stats(v) for ph, v in samples.items()},
                     "workgroup_start": stats(starts), "workgroup_end": stats(ends),
                     "span_first_start_to_last_end": stats(spans)}
    print(json.dumps(out), flush=True)


READ_PROBE_SRC = r"""
#include <hip/hip_runtime.h>
// Plain reads of rows x v floats with non-temporal 16-byte loads; one float per workgroup is
// written so that the loads are kept.
//   rows_read:   one 1024-thread workgroup per row, one load per lane and step
//   rows_chunks: one 1024-thread workgroup per row in the verification's order (wave w takes
//                1024-float chunks w, w + 16, ..., four loads per lane and chunk)
//   rows_split:  S workgroups of T threads per row, each a contiguous share, four loads per lane
//   grid_read:   a grid-stride loop over the whole array, 2,048 workgroups of 256 threads
typedef float f4v __attribute__((ext_vector_type(4)));
__global__ void __launch_bounds__(1024) rows_read(const float *x, long v, float *out) {
    const f4v *r = reinterpret_cast<const f4v *>(x + (long)blockIdx.x * v);
    const long n4 = v / 4;
    f4v acc = {0, 0, 0, 0};
    for (long k = threadIdx.x; k < n4; k += 1024) acc += __builtin_nontemporal_load(r + k);
    const float s = acc.x + acc.y + acc.z + acc.w;
    if (s == 12345.0f) out[blockIdx.x] = s;
}
__global__ void __launch_bounds__(1024) rows_chunks(const float *x, long v, float *out) {
    const f4v *r = reinterpret_cast<const f4v *>(x + (long)blockIdx.x * v);
    const int lane = threadIdx.x % 64, wave = threadIdx.x / 64;
    const long n4 = v / 4;
    f4v acc = {0, 0, 0, 0};
    for (long c = wave; c * 256 < n4; c += 16) {
        f4v t[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
            const long k = c * 256 + u * 64 + lane;
            t[u] = k < n4 ? __builtin_nontemporal_load(r + k) : f4v{0, 0, 0, 0};
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) acc += t[u];
    }
    const float s = acc.x + acc.y + acc.z + acc.w;
    if (s == 12345.0f) out[blockIdx.x] = s;
}
template <int T>
__global__ void __launch_bounds__(T) rows_split(const float *x, long v, int S, float *out) {
    const int b = blockIdx.x / S, s = blockIdx.x % S;
    const long n4 = v / 4, lo = n4 * s / S, hi = n4 * (s + 1) / S;
    const f4v *r = reinterpret_cast<const f4v *>(x + (long)b * v);
    f4v acc = {0, 0, 0, 0};
    long k = lo + threadIdx.x;
    for (; k + 3 * T < hi; k += 4 * T) {
        f4v t[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) t[u] = __builtin_nontemporal_load(r + k + u * T);
#pragma unroll
        for (int u = 0; u < 4; ++u) acc += t[u];
    }
    for (; k < hi; k += T) acc += __builtin_nontemporal_load(r + k);
    const float sm = acc.x + acc.y + acc.z + acc.w;
    if (sm == 12345.0f) out[blockIdx.x % 4096] = sm;
}
__global__ void __launch_bounds__(256) grid_read(const float *x, long n4, float *out) {
    const f4v *r = reinterpret_cast<const f4v *>(x);
    f4v acc = {0, 0, 0, 0};
    for (long k = blockIdx.x * 256L + threadIdx.x; k < n4; k += (long)gridDim.x * 256) acc += __builtin_nontemporal_load(r + k);
    const float s = acc.x + acc.y + acc.z + acc.w;
    if (s == 12345.0f) out[blockIdx.x] = s;
}
// kind 0: rows_read, 1: rows_chunks, 2: rows_split 2 x 512, 3: rows_split 4 x 256, 4: grid_read
extern "C" int probe(int kind, const float *x, int rows, long v, float *out, void *stream) {
    hipStream_t st = (hipStream_t)stream;
    switch (kind) {
    case 0: hipLaunchKernelGGL(rows_read, dim3(rows), dim3(1024), 0, st, x, v, out); break;
    case 1: hipLaunchKernelGGL(rows_chunks, dim3(rows), dim3(1024), 0, st, x, v, out); break;
    case 2: hipLaunchKernelGGL(rows_split<512>, dim3(rows * 2), dim3(512), 0, st, x, v, 2, out); break;
    case 3: hipLaunchKernelGGL(rows_split<256>, dim3(rows * 4), dim3(256), 0, st, x, v, 4, out); break;
    case 4: hipLaunchKernelGGL(grid_read, dim3(2048), dim3(256), 0, st, x, (long)rows * v / 4, out); break;
    default: return 2;
    }
    return hipGetLastError() == hipSuccess ? 0 : 1;
}
"""


def main_read_ceiling(args):
    """Plain reads of the verification's row bytes (256 rows x 151,936 fp32, one replica of four
    per launch, as the benchmark rotates them), by read-only kernels built here from the source
    above: the verification's launch shape (a 1024-thread workgroup per row, also in its chunk
    order), several workgroups per row, and a grid-stride loop; for reference torch.sum of the
    same bytes and a device-to-device copy.  The kernels run eight to a HIP graph; torch.sum and the
    copy are launched back to back (no graph: the library reduction may clear its scratch with
    memsets); HIP events."""
    import subprocess
    import tempfile

    import torch

    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    rows, v = 256, 151_936
    tmp = tempfile.mkdtemp(prefix="tt_read_probe_")
    src, lib = os.path.join(tmp, "probe.hip"), os.path.join(tmp, "probe.so")
    with open(src, "w") as f:
        f.write(READ_PROBE_SRC)
    subprocess.run(["/opt/rocm/bin/hipcc", "--offload-arch=gfx950", "-O3", "-fPIC", "-shared", "-Xclang",
                    "-target-feature", "-Xclang", "-packed-fp32-ops", src, "-o", lib], check=True,
                   stdout=subprocess.DEVNULL, stderr=subprocess.DEVNULL)
    P = ctypes.CDLL(lib)
    P.probe.argtypes = [ctypes.c_int, ctypes.c_void_p, ctypes.c_int, ctypes.c_long, ctypes.c_void_p, ctypes.c_void_p]
    R = max(1, args.replicas)
    g = torch.Generator(device=dev)
    g.manual_seed(5005)
    xs = [torch.rand((rows, v), generator=g, device=dev) for _ in range(R)]
    dst = torch.empty_like(xs[0])
    sink = torch.zeros(4096, device=dev)
    nbytes = 4 * rows * v
    reps = max(8, args.steps)

    def stream():
        return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)

    kinds = {"rows_read": 0, "rows_chunks": 1, "rows_split_2x512": 2, "rows_split_4x256": 3, "grid_read": 4}
    probe_ms = {name: graph_ms(lambda i, kd=kd: P.probe(kd, xs[i % R].data_ptr(), rows, v, sink.data_ptr(), stream()),
                               k=8, reps=max(2, reps // 8)) for name, kd in kinds.items()}

    def eager_ms(fn):
        for i in range(4):
            fn(i)
        torch.cuda.synchronize()
        s0, s1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        s0.record()
        for i in range(reps):
            fn(i)
        s1.record()
        torch.cuda.synchronize()
        return s0.elapsed_time(s1) / reps

    sum_ms = eager_ms(lambda i: torch.sum(xs[i % R]))
    copy_ms = eager_ms(lambda i: dst.copy_(xs[i % R]))

    def gbs(ms, k=1):
        return round(k * nbytes / (ms * 1e-3) / 1e9, 1)

    out = {"metric": "plain HBM reads of the benchmark's row bytes", "bytes_per_launch": nbytes}
    for name, ms in probe_ms.items():
        out[name + "_us"] = round(ms * 1e3, 2)
        out[name + "_GBps"] = gbs(ms)
    out.update({"torch_sum_us": round(sum_ms * 1e3, 2), "torch_sum_GBps": gbs(sum_ms),
                "copy_us": round(copy_ms * 1e3, 2), "copy_read_write_GBps": gbs(copy_ms, 2),
                "peak_GBps": HBM_PEAK_GBS})
    print(json.dumps(out), flush=True)


def tli_workload(dev, n, M):
    """The TLI benchmark's inputs, generated on the GPU (seeded): the intersection of the
    benchmark's vocabularies, n streams x M draft rows softmax(3 N(0,1)) over V_d, proposals
    drawn from q', target rows softmax(3 N(0,1)) over V_t with the proposal raised to the row's
    maximum + 1 at half of the positions, the drafter's masses S_j (fp32 sums), uniforms on
    the 2^-24 grid."""
    import torch

    import paper_2510_15545_amd as tt
    from paper_2510_15545_amd import synth

    S = synth.make(3, n_streams=4, probs=False)
    vd = tt.Vocab.from_host(S.vocab_d.data, S.vocab_d.offsets, S.vocab_d.max_len, dev)
    vt = tt.Vocab.from_host(S.vocab_t.data, S.vocab_t.offsets, S.vocab_t.max_len, dev)
    d2t, t2d = tt.vocab_intersection(vd, tt.token_index(vd), vt, tt.token_index(vt))
    v_d, v_t = int(d2t.numel()), int(t2d.numel())
    nt = n * M
    g = torch.Generator(device=dev)
    g.manual_seed(4004)
    q = torch.softmax(torch.randn((nt, v_d), generator=g, device=dev).mul_(3.0), dim=1)
    qp = tt.tli_proposal(d2t, t2d, q)
    ys = torch.multinomial(qp, 1, generator=g).view(-1).to(torch.int32)
    del qp
    off = torch.arange(0, nt + 1, M, dtype=torch.int32, device=dev)
    x = torch.randn((nt + n, v_t), generator=g, device=dev).mul_(3.0)
    rows = (torch.arange(nt, device=dev) // M) * (M + 1) + torch.arange(nt, device=dev) % M
    force = torch.rand(nt, generator=g, device=dev) < 0.5
    x[rows[force], ys.long()[force]] = x[rows[force]].max(dim=1).values + 1.0
    p = torch.softmax(x, dim=1)
    del x
    mass = (q * (d2t >= 0).to(torch.float32)).sum(dim=1).contiguous()
    ua = torch.randint(0, 1 << 24, (nt,), generator=g, device=dev).float().mul_(2.0 ** -24)
    us = torch.randint(0, 1 << 24, (n,), generator=g, device=dev).float().mul_(2.0 ** -24)
    return {"d2t": d2t, "t2d": t2d, "ys": ys, "off": off, "q": q, "p": p, "mass": mass, "ua": ua, "us": us,
            "n": n, "M": M, "nt": nt, "v_d": v_d, "v_t": v_t, "inter": int((d2t >= 0).sum().item())}


def main_tli(args):
    """TLI verification (App. D Alg. 3 feeding Alg. 4): 256 streams x M=8 drafted positions over
    the benchmark's vocabularies (V_d 128,256, V_t 151,936, their byte-string intersection);
    draft rows softmax(3 N(0,1)), proposals drawn from q', target rows softmax(3 N(0,1)) with
    the proposal raised to the row's maximum + 1 at half of the positions.  Inputs are generated
    on the GPU (seeded).  Timed: tt_verify_tli with the drafter's masses (the step), without
    them, and tt_tli_proposal over every draft row followed by tt_verify_dense."""
    import torch

    import paper_2510_15545_amd as tt

    tt.lib()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    t_gen = time.time()
    W = tli_workload(dev, args.streams or 256, 8)
    d2t, t2d, ys, off, q, p, mass, ua, us = (W[k] for k in ("d2t", "t2d", "ys", "off", "q", "p", "mass", "ua", "us"))
    # consecutive steps read different copies of the draft and target rows (as in the default
    # benchmark), so the Infinity Cache cannot serve a step from the one before
    R = max(1, args.replicas)
    qs, ps = [q], [p]
    for _ in range(R - 1):
        qs.append(q.clone())
        ps.append(p.clone())
    n, M, nt, v_t, inter = W["n"], W["M"], W["nt"], W["v_t"], W["inter"]
    v_d = W["v_d"]
    torch.cuda.synchronize()
    t_gen = time.time() - t_gen
    nacc = torch.empty(n, dtype=torch.int32, device=dev)
    tok = torch.empty(n, dtype=torch.int32, device=dev)
    outs = {}

    def fused(with_mass):
        return lambda i: tt.verify_tli(d2t, t2d, ys, off, qs[i % R], ps[i % R], ua, us, M,
                                       draft_mass=mass if with_mass else None, out=(nacc, tok))
    qbuf = torch.empty((nt, v_t), dtype=torch.float32, device=dev)
    ws = tt.verify_workspace(n, v_t, dev)

    def two_calls(i):
        tt.tli_proposal(d2t, t2d, qs[i % R], out=qbuf)
        tt.verify_dense(v_t, ys, off, qbuf, ps[i % R], ua, us, M, workspace=ws, out=(nacc, tok, None))

    times = {}
    # --eager (profiler passes): only the fused call with the drafter's masses, launched one by one
    runs = (("fused_with_mass", fused(True)),) if args.eager else \
        (("fused_with_mass", fused(True)), ("fused", fused(False)), ("two_calls", two_calls))
    for name, fn in runs:
        fn(0)
        torch.cuda.synchronize()
        outs[name] = (nacc.cpu().numpy().copy(), tok.cpu().numpy().copy())
        if args.eager:
            reps = max(2, args.steps)
            s0, s1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            s0.record()
            for i in range(reps):
                fn(i)
            s1.record()
            torch.cuda.synchronize()
            times[name] = s0.elapsed_time(s1) / reps
        else:
            times[name] = graph_ms(fn, k=max(1, min(args.graph_steps, 8)), reps=max(2, args.steps // 8))
    copy_calibration(args, dev)
    if "fused" not in outs:
        outs["fused"] = outs["fused_with_mass"]
    # the drafter's S here is an fp32 sum, not the exact intersected mass the kernel forms without
    # it, so that run is compared with the others only through its acceptance counts
    acc = outs["fused"][0]
    tested = int(np.minimum(acc + 1, M).sum())
    rejected = int((acc < M).sum())
    ms = times["fused_with_mass"]
    # algorithmic bytes with the drafter's masses: per tested position the id, u, S, t2d entry,
    # gathered draft mass and target probability; per stream the target row gamma, u_sample and
    # the outputs; per rejected stream the draft masses on the intersection; the map t2d once
    kbytes = int(24 * tested + n * (4 * v_t + 12) + rejected * 4 * inter + 4 * v_t)
    gbs = kbytes / (ms * 1e-3) / 1e9
    acc_m = outs["fused_with_mass"][0]
    wl_name = f"{n} streams x M={M}, V_d={v_d}, V_t={v_t}, intersection {inter}"
    traffic, note = read_traffic(args.traffic or os.path.join(ROOT, "profiles", "verify_tli_row_counters.txt"),
                                 wl_name, "verify_tli_row")
    result = {
        "metric": "verified draft tokens/s, TLI proposals (App. D Alg. 3 + 4) at V_d=128,256 / V_t=151,936; "
                  "HBM GB/s vs peak",
        "value": round(nt / (ms * 1e-3), 1), "unit": "draft tokens/s", "n_gpus": 1,
        "steps": max(2, args.steps // 8) * max(1, min(args.graph_steps, 8)), "warmup": 1,
        "ms_per_step": round(ms, 5), "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f32+i64", "data": "synthetic",
        "config": {"workload": wl_name, "streams": n,
                   "draft_tokens_per_step": nt, "path": "tt_verify_tli with the drafter's masses", "replicas": R,
                   "launch": "eager" if args.eager else "hip-graph of %d steps" % max(1, min(args.graph_steps, 8))},
        "accept": {"mean_gamma": round(float(acc_m.mean()), 3), "rejected_streams": int((acc_m < M).sum())},
        "us_per_step": {k: round(v * 1e3, 2) for k, v in times.items()},
        "same_outputs_fused_and_two_calls": None if "two_calls" not in outs else bool(
            np.array_equal(outs["fused"][0], outs["two_calls"][0]) and
            np.array_equal(outs["fused"][1], outs["two_calls"][1])),
        "with_mass_acceptance_agreement": round(float((acc_m == acc).mean()), 4),
        "roofline": {"kernel": "verify_tli_row", "bound": "hbm", "achieved": round(gbs, 1), "peak": HBM_PEAK_GBS,
                     "unit": "GB/s", "frac": round(gbs / HBM_PEAK_GBS, 4), "traffic": traffic,
                     "traffic_note": note, "algorithmic_bytes_per_launch": kbytes,
                     "launch_us": round(ms * 1e3, 2)},
        "gen_seconds": round(t_gen, 1),
    }
    print(json.dumps(result), flush=True)


def main_logits(args):
    """Verification from bf16 logits (tt_verify_logits) on the benchmark's streams: the same
    target ids, offsets and uniforms, target logits bf16(3 N(0,1)) with the logit of each
    proposal raised to the row's maximum + 1 at 30% of the positions, temperature 0.7, proposal
    masses uniform in [0.05, 0.55).  Logits are generated on the GPU (seeded) and replicated
    like the probability rows."""
    import torch

    import paper_2510_15545_amd as tt
    from paper_2510_15545_amd import synth

    tt.lib()
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    t_gen = time.time()
    S = synth.make(3, n_streams=args.streams, probs=False)
    n, V = S.n, S.v_t
    m = np.diff(S.target_off)
    rows = int(S.target_off[-1]) + n
    g = torch.Generator(device=dev)
    g.manual_seed(3003)
    x = torch.randn((rows, V), generator=g, device=dev, dtype=torch.float32).mul_(3.0)
    row_of = torch.from_numpy((S.target_off[:-1] + np.arange(n))[np.repeat(np.arange(n), m)] +
                              (np.arange(int(m.sum())) - np.repeat(S.target_off[:-1], m))).to(dev).long()
    ids_l = torch.from_numpy(S.verify_ids.astype(np.int64)).to(dev)
    force = torch.rand(int(m.sum()), generator=g, device=dev) < 0.3
    x[row_of[force], ids_l[force]] = x[row_of[force]].max(dim=1).values + 1.0
    R = max(1, args.replicas)
    logits = [x.to(torch.bfloat16)]
    del x
    for _ in range(R - 1):
        logits.append(logits[0].clone())
    q = (torch.rand(int(m.sum()), generator=g, device=dev) * 0.5 + 0.05).contiguous()
    it = torch.full((n,), 1.0 / 0.7, dtype=torch.float32, device=dev)

    def t(a):
        return torch.from_numpy(np.ascontiguousarray(a)).to(dev)

    ids, off = t(S.verify_ids), t(S.target_off)
    # uniforms on the 2^-24 grid, as the generator draws them
    ua = torch.randint(0, 1 << 24, (int(m.sum()),), generator=g, device=dev).float().mul_(2.0 ** -24)
    us = torch.randint(0, 1 << 24, (n,), generator=g, device=dev).float().mul_(2.0 ** -24)
    max_m = max(1, int(m.max()))
    nacc = torch.empty(n, dtype=torch.int32, device=dev)
    tok = torch.empty(n, dtype=torch.int32, device=dev)
    lse = None
    if args.lse:  # what an LM head would emit with its logits: log-sum-exp of logit / T per row
        row_it = it.repeat_interleave(torch.from_numpy(m + 1).to(dev))
        lse = torch.cat([(logits[0][i:i + 256].float() * row_it[i:i + 256, None]).logsumexp(dim=1)
                         for i in range(0, rows, 256)]).contiguous()
    torch.cuda.synchronize()
    t_gen = time.time() - t_gen

    def step(r):
        tt.verify_logits(V, ids, off, q, logits[r], it, ua, us, max_m, lse=lse, out=(nacc, tok))

    for i in range(args.warmup):
        step(i % R)
    torch.cuda.synchronize()
    gs = 1 if args.eager else max(1, min(args.graph_steps, args.steps))
    reps = max(1, args.steps // gs)
    s0, s1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    if args.eager:
        s0.record()
        for i in range(reps):
            step(i % R)
        s1.record()
    else:
        gr = torch.cuda.CUDAGraph()
        cap = torch.cuda.Stream()
        cap.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(cap):
            with torch.cuda.graph(gr, stream=cap):
                for i in range(gs):
                    step(i % R)
        torch.cuda.current_stream().wait_stream(cap)
        gr.replay()
        torch.cuda.synchronize()
        s0.record()
        for _ in range(reps):
            gr.replay()
        s1.record()
    torch.cuda.synchronize()
    ms = s0.elapsed_time(s1) / (reps * gs)
    step(0)
    torch.cuda.synchronize()
    copy_calibration(args, dev)
    acc = nacc.cpu().numpy()
    if lse is None:
        # algorithmic bytes: each row a stream reads (rows 0 .. gamma, once), t_j, q_j, u_j per
        # position, 1/T, u_sample, n_accepted, out_token
        rows_read = int((np.minimum(acc, m) + 1).sum())
        kbytes = int(2 * V * rows_read + 12 * int(m.sum()) + 16 * n)
    else:
        # one row per stream (the residual or bonus row) and its L; per position tested
        # (0 .. min(gamma, M - 1)) t_j, q_j, u_j, L_j and the gathered logit
        rows_read = n
        tested = int(np.minimum(acc + 1, m).sum())
        kbytes = int(2 * V * n + 4 * n + 18 * tested + 16 * n)
    gbs = kbytes / (ms * 1e-3) / 1e9
    elems_per_s = V * rows_read / (ms * 1e-3)
    draft_tokens = int(S.draft_off[-1])
    wl_name = f"{n} streams V_t={V} bf16 logits T=0.7 30% forced" + (" with row log-sum-exp" if lse is not None else "")
    traffic, note = read_traffic(args.traffic or os.path.join(
        ROOT, "profiles", "verify_logits_row" + ("_lse" if lse is not None else "") + "_counters.txt"),
        wl_name, "verify_logits_row")
    result = {
        "metric": "verified draft tokens/s from bf16 logits (T=0.7) at V_t=151,936; HBM GB/s vs peak",
        "value": round(draft_tokens / (ms * 1e-3), 1), "unit": "draft tokens/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 5), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "bf16+f32+i64", "data": "synthetic",
        "config": {"workload": wl_name, "streams": n,
                   "target_positions": int(m.sum()), "v_t": V, "replicas": R, "path": "tt_verify_logits" + ("+lse" if lse is not None else ""),
                   "launch": "eager" if args.eager else "hip-graph of %d steps" % gs},
        "accept": {"mean_gamma": round(float(acc.mean()), 3), "rows_read": rows_read},
        "roofline": {"kernel": "verify_logits_row", "bound": "hbm", "achieved": round(gbs, 1),
                     "peak": HBM_PEAK_GBS, "unit": "GB/s", "frac": round(gbs / HBM_PEAK_GBS, 4), "traffic": traffic,
                     "traffic_note": note, "algorithmic_bytes_per_launch": kbytes,
                     "launch_us": round(ms * 1e3, 2), "logits_per_s": round(elems_per_s, 1)},
        "gen_seconds": round(t_gen, 1),
    }
    print(json.dumps(result), flush=True)


def synth_fits_fused(S):
    """The fused kernel's shape conditions (mirrors the library's dispatch rule)."""
    nc = (S.v_t + 1023) // 1024
    return S.max_k <= 64 and S.max_m <= 64 and ((S.n >= 256 and nc <= 2048) or S.v_t <= 16384)


def graph_ms(fn, k=20, reps=10):
    """ms per call: k calls captured in one HIP graph, replayed `reps` times, HIP events on the
    stream the graph runs on."""
    import torch

    g = torch.cuda.CUDAGraph()
    cap = torch.cuda.Stream()
    cap.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(cap):
        with torch.cuda.graph(g, stream=cap):
            for i in range(k):
                fn(i)
    torch.cuda.current_stream().wait_stream(cap)
    g.replay()
    torch.cuda.synchronize()
    s0, s1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    s0.record()
    for _ in range(reps):
        g.replay()
    s1.record()
    torch.cuda.synchronize()
    return s0.elapsed_time(s1) / (k * reps)


def acceptance(nacc, target_off):
    """Acceptance of a verified batch: accepted / proposed positions (sum gamma / sum M), accepted /
    tested positions (a stream tests positions up to and including its first rejection), the
    share of streams accepting at least one position and the mean gamma."""
    g = np.asarray(nacc, np.int64)
    M = np.diff(np.asarray(target_off, np.int64))
    ok = g >= 0
    g, M = g[ok], M[ok]
    tested = np.minimum(g + 1, M)
    return {"accept_rate": round(float(g.sum()) / max(1, int(M.sum())), 4),
            "per_position_accept_rate": round(float(g.sum()) / max(1, int(tested.sum())), 4),
            "streams_with_gamma_above_0": round(float((g > 0).mean()) if g.size else 0.0, 4),
            "mean_gamma": round(float(g.mean()) if g.size else 0.0, 3)}


def dtw_stress(dev, w):
    """The DTW stress batch (workload 4: 1,024 pairs of 64-512 tokens each side) through tt_align,
    with the strip kernel's VALU issue fraction and LDS bank-conflict rate from the counter
    summary (when it covers the current kernel sources)."""
    import torch

    import paper_2510_15545_amd as tt
    from paper_2510_15545_amd import synth

    t0 = time.time()
    wl = synth.make(4, probs=False, w=w)
    gen = time.time() - t0
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)  # noqa: E731
    vd = tt.Vocab.from_host(wl.vocab_d.data, wl.vocab_d.offsets, wl.vocab_d.max_len, dev)
    vt = tt.Vocab.from_host(wl.vocab_t.data, wl.vocab_t.offsets, wl.vocab_t.max_len, dev)
    di, do, ti, to = t(wl.draft_ids), t(wl.draft_off), t(wl.target_ids), t(wl.target_off)
    mtb = max(wl.vocab_d.max_len, wl.vocab_t.max_len)
    ws = tt.align_workspace(wl.n, wl.max_k, wl.max_m, w, mtb, dev)
    out = tt.align(vd, vt, di, do, ti, to, w, wl.max_k, wl.max_m,
                   n_path=tt.path_capacity(wl.draft_off[-1], wl.target_off[-1]), workspace=ws)
    torch.cuda.synchronize()
    ms = graph_ms(lambda i: tt.align(vd, vt, di, do, ti, to, w, wl.max_k, wl.max_m, out=out, workspace=ws),
                  k=10, reps=5)
    K, M = np.diff(wl.draft_off), np.diff(wl.target_off)
    cells = band_cells(K, M, w)
    # the step before the alignment on the same pairs: draft ids -> proxy target ids (greedy
    # longest match); the token index is built once, outside the timing
    idx = tt.token_index(vt)
    maxb = int(max(np.add.reduceat(np.diff(wl.vocab_d.offsets)[wl.draft_ids], wl.draft_off[:-1])))
    rt = (torch.empty(wl.n * wl.max_m, dtype=torch.int32, device=dev), torch.empty(wl.n + 1, dtype=torch.int32, device=dev))
    tt.retokenize(vd, vt, idx, di, do, maxb, wl.max_m, out=rt)
    torch.cuda.synchronize()
    rt_ok = bool(np.array_equal(rt[1].cpu().numpy(), wl.target_off) and
                 np.array_equal(rt[0].cpu().numpy()[:int(wl.target_off[-1])], wl.target_ids))
    ms_rt = graph_ms(lambda i: tt.retokenize(vd, vt, idx, di, do, maxb, wl.max_m, out=rt), k=10, reps=5)
    kv, why = read_counters(os.path.join(ROOT, "profiles", "dtw_band_counters.txt"), wl.spec.name, "dtw_band")
    issue = None
    if kv is not None:  # wave instructions over the 1,024 SIMDs' issue slots (one per 4 cycles)
        issue = int(kv["valu_instructions_per_launch"]) / (256 * 4 * 2.4e9 / 4 * ms * 1e-3)
    return {"workload": wl.spec.name, "pairs": wl.n, "w": w, "tt_align_us": round(ms * 1e3, 2),
            "band_cells": cells, "band_cells_per_s": round(cells / (ms * 1e-3), 1),
            "full_cells_per_s": round(int((K * M).sum()) / (ms * 1e-3), 1),
            "valu_issue_frac": None if issue is None else round(issue, 4),
            "lds_bank_conflict_rate": None if kv is None else float(kv["lds_bank_conflict_rate"]),
            "counter_note": why or "dtw_band SQ_INSTS_VALU per launch over the tt_align call's time",
            "tt_retokenize_us": round(ms_rt * 1e3, 2),
            "retokenize_bytes": int((np.diff(wl.vocab_d.offsets)[wl.draft_ids]).sum()),
            "retokenize_matches_workload": rt_ok,
            "gen_seconds": round(gen, 1)}


def high_acceptance(dev, args, R):
    """The benchmark batch with leading runs of forced positions instead of independent ones
    (synth force_runs = 0.9): most streams accept several positions, so the rows after the
    first position are the ones streamed.  One tt_step per step, and tt_verify alone."""
    import torch

    import paper_2510_15545_amd as tt
    from paper_2510_15545_amd import synth

    S = synth.make(3, w=args.w, force_runs=0.9)
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a)).to(dev)  # noqa: E731
    vd = tt.Vocab.from_host(S.vocab_d.data, S.vocab_d.offsets, S.vocab_d.max_len, dev)
    vt = tt.Vocab.from_host(S.vocab_t.data, S.vocab_t.offsets, S.vocab_t.max_len, dev)
    di, do, ti, to = t(S.draft_ids), t(S.draft_off), t(S.target_ids), t(S.target_off)
    dp = t(S.draft_probs)
    rows = [t(S.target_probs)]
    for _ in range(R - 1):
        rows.append(rows[0].clone())
    ua, us = t(S.u_accept), t(S.u_sample)
    n, mtb = S.n, max(S.vocab_d.max_len, S.vocab_t.max_len)
    st_ws = tt.step_workspace(n, S.v_t, S.max_k, S.max_m, args.w, mtb, dev)
    out = tt.step(vd, vt, S.v_d, S.v_t, di, do, ti, to, args.w, S.max_k, S.max_m, dp, rows[0], ua, us,
                  workspace=st_ws)
    step = lambda i: tt.step(vd, vt, S.v_d, S.v_t, di, do, ti, to, args.w, S.max_k, S.max_m, dp,  # noqa: E731
                             rows[i % R], ua, us, workspace=st_ws, out=out)
    ms_step = graph_ms(step, k=8, reps=10)
    q = out[4]
    ws = tt.verify_workspace(n, S.v_t, dev)
    vo = (torch.empty(n, dtype=torch.int32, device=dev), torch.empty(n, dtype=torch.int32, device=dev), None)
    ms_verify = graph_ms(lambda i: tt.verify(S.v_t, ti, to, q, rows[i % R], ua, us, S.max_m, workspace=ws, out=vo))
    torch.cuda.synchronize()
    m = np.diff(S.target_off)
    vbytes = int(n * 4 * S.v_t + 16 * int(m.sum()) + 12 * n)
    res = {"workload": S.spec.name.replace("30% forced", "forced leading runs (p 0.9)"),
           "ms_per_step": round(ms_step, 5), "draft_tokens_per_s": round(int(S.draft_off[-1]) / (ms_step * 1e-3), 1),
           "verify_us": round(ms_verify * 1e3, 2),
           "verify_frac_of_peak": round(vbytes / (ms_verify * 1e-3) / 1e9 / HBM_PEAK_GBS, 4)}
    res.update(acceptance(out[5].cpu().numpy(), S.target_off))
    return res


def cpu_baseline(args, S, A, nacc, tok, s_out, a_out):
    """The oracle, unmodified, on the host cores: whole steps over the same batch,
    repeated until about --cpu-seconds of work; also checks the GPU outputs."""
    import oracle

    threads = len(os.sched_getaffinity(0))
    reps, t0 = 0, time.time()
    out = None
    while reps == 0 or time.time() - t0 < args.cpu_seconds:
        if S is not A:
            oracle.align(A.vocab_d.data, A.vocab_d.offsets, A.vocab_d.max_len, A.vocab_t.data,
                         A.vocab_t.offsets, A.vocab_t.max_len, A.draft_ids, A.draft_off, A.target_ids,
                         A.target_off, args.w, n_threads=threads)
        out = oracle.run_workload(S, n_threads=threads)
        reps += 1
    dt = (time.time() - t0) / reps
    # the same on one thread, for a third of the time
    reps1, t1 = 0, time.time()
    while reps1 == 0 or time.time() - t1 < args.cpu_seconds / 3:
        if S is not A:
            oracle.align(A.vocab_d.data, A.vocab_d.offsets, A.vocab_d.max_len, A.vocab_t.data,
                         A.vocab_t.offsets, A.vocab_t.max_len, A.draft_ids, A.draft_off, A.target_ids,
                         A.target_off, args.w, n_threads=1)
        oracle.run_workload(S, n_threads=1)
        reps1 += 1
    dt1 = (time.time() - t1) / reps1
    draft_tokens = int(S.draft_off[-1])
    match = bool(np.array_equal(out["n_accepted"], nacc.cpu().numpy()) and
                 np.array_equal(out["out_token"], tok.cpu().numpy()) and
                 np.array_equal(out["cost"], s_out[0].cpu().numpy()))
    return {"value": round(draft_tokens / dt, 1), "unit": "draft tokens/s", "cores": threads,
            "kind": "oracle", "sample": f"{reps} whole steps of the benchmark batch "
                                        f"({S.n} streams), {dt * 1e3:.1f} ms each",
            "value_1_thread": round(draft_tokens / dt1, 1),
            "sample_1_thread": f"{reps1} whole steps, {dt1 * 1e3:.1f} ms each",
            "cpu_model": cpu_model(), "matches_gpu": match}


def cpu_model():
    """The host CPU's model name (/proc/cpuinfo), or None."""
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


if __name__ == "__main__":
    main()
