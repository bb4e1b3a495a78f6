#!/usr/bin/env python3
"""Benchmark of the stacked-prompt prefill attention on one MI355X.

For each workload, one prefill call computes the attention output of every
header token (every instruction, context and question token of every
prompt) for one layer; ippd_prefill_attention serves all question tokens of
a prompt from one pass over its context and computes the context rows once,
standard_prefill_attention prefills each question's own prompt
[context; question] (Sec. 3, standard prompting).  Both run on identical
caches and queries; the timed region is R calls back to back on one stream
(HIP events on that stream), after W warmup calls (and, before the first
path, at least 200 ms of untimed calls while the clocks ramp up).

Reported per workload (one JSON line each):
  value        header tokens per second of the IPPD call (sum of context and
               question tokens / seconds per call);
  roofline     bound "mfma": algorithmic FLOPs of one call (4*D per visible
               (row, key) pair and query head: Q.K and P.V) / its time,
               against the dense bf16 MFMA peak of 2500 TFLOP/s;
  standard     the baseline's time, its FLOPs (the context rows recomputed
               once per question) and the IPPD speedup;
  folded_one_level  (two-level workloads) the IPPD prefill of the same prompts
               as a one-level batch, each context carrying its own copy of
               the instruction;

Usage: python bench_prefill.py [--workload NAME|all] [--reps 30] [--warmup 30]
       python bench_prefill.py --sweep questions|context
The sweeps are the prefill analogue of the paper's ablations (App. D): one
Llama-3-8B-shaped prompt with questions of 32 tokens, N = 1..32 questions at
context 4096, or context 1024..8192 at N = 16; one line per point, then a
markdown table of the IPPD and standard times.
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import workload as W  # noqa: E402

MFMA_BF16_PEAK_TFLOPS = 2500.0
MFMA_F32_PEAK_TFLOPS = 157.3

WORKLOADS = {
    # Llama-3-8B attention shape, one prompt: context 4096, 16 questions of 32 tokens.
    "llama3-8b-lc4096-n16-q32": dict(wid=500, num_prompts=1, ctx_len=(4096, 4096), questions=(16, 16),
                                     question_tokens=32, seg_len=(0, 0)),
    # NarrativeQA-like shape (shared context ~3.5k tokens, ~30 questions of ~12 tokens).
    "narrativeqa-shape-lc3500-n30-q12": dict(wid=501, num_prompts=1, ctx_len=(3500, 3500), questions=(30, 30),
                                             question_tokens=12, seg_len=(0, 0)),
    # 8 ragged prompts: context U{1024..8192}, 4..32 questions of U{8..32} tokens.
    "ragged-b8": dict(wid=502, num_prompts=8, ctx_len=(1024, 8192), questions=(4, 32), question_tokens=0,
                      seg_len=(8, 32)),
    # two-level (Sec. 4.4): 8 contexts of 1024 tokens behind 2 instructions of
    # 2048 tokens (4 contexts each), 8 questions of 16 tokens per context.
    "two-level-b8-cpi4-lp2048": dict(wid=503, num_prompts=8, ctx_len=(1024, 1024), questions=(8, 8),
                                     question_tokens=16, seg_len=(0, 0), instr=(4, (2048, 2048))),
}


SWEEP_QUESTIONS = [1, 2, 4, 8, 16, 32]            # at context 4096
SWEEP_CONTEXT = [1024, 2048, 4096, 8192]           # at N = 16


def sweep_points(kind: str):
    pts = [(n, 4096) for n in SWEEP_QUESTIONS] if kind == "questions" else [(16, lc) for lc in SWEEP_CONTEXT]
    names = []
    for n, lc in pts:
        name = f"sweep-n{n}-lc{lc}"
        WORKLOADS[name] = dict(wid=520 + n + lc // 256, num_prompts=1, ctx_len=(lc, lc), questions=(n, n),
                               question_tokens=32, seg_len=(0, 0))
        names.append((name, n, lc))
    return names


def make(name: str) -> W.DecodeWorkload:
    kw = {k: v for k, v in WORKLOADS[name].items() if k != "instr"}
    return W.custom_workload(name=name, dtype="bf16", hq=32, hkv=8, head_dim=128, steps=1, value_std=0.5, **kw)


def flops(st: W.Structure, standard: bool, ins=None) -> float:
    """Algorithmic FLOPs of one call: 4*D*Hq per visible (query row, key) pair.
    The baseline computes the rows of an instruction and of a context once per
    question whose prompt holds them, IPPD once."""
    wl = st.wl
    per = 4.0 * wl.head_dim * wl.hq
    tot = 0.0
    s_of = (np.searchsorted(ins.prompt_start, np.arange(wl.num_prompts), side="right") - 1
            if ins is not None else None)
    if ins is not None:
        for s_ in range(len(ins.lp)):
            lp = int(ins.lp[s_])
            nq = int(st.q_start[ins.prompt_start[s_ + 1]] - st.q_start[ins.prompt_start[s_]])
            tot += per * lp * (lp + 1) / 2 * (nq if standard else 1)
    for b in range(wl.num_prompts):
        lc = int(st.ctx_len[b])
        lp = int(ins.lp[s_of[b]]) if ins is not None else 0
        qs = range(int(st.q_start[b]), int(st.q_start[b + 1]))
        ctx_pairs = lc * lp + lc * (lc + 1) / 2
        tot += per * ctx_pairs * (len(qs) if standard else 1)   # context rows: once per question / once
        for i in qs:
            s = int(st.seg_len0[i])
            tot += per * (s * (lp + lc) + s * (s + 1) / 2)
    return tot


def folded_time(st, kv, pq, ins, iq, reps: int, warmup: int) -> float:
    """IPPD prefill of the one-level batch in which context b is [p_s; c_b]
    (the instruction copied into every context behind it)."""
    import torch
    from paper_2609_05707_amd.session import DecodeBatch
    wl = st.wl
    s_of = np.searchsorted(ins.prompt_start, np.arange(wl.num_prompts), side="right") - 1
    fk, fv, fq, flen = [], [], [], []
    for b in range(wl.num_prompts):
        i0, i1 = ins.tok_start[s_of[b]], ins.tok_start[s_of[b] + 1]
        c0, c1 = st.ctx_start[b], st.ctx_start[b + 1]
        fk.append(np.concatenate([ins.k[i0:i1], kv.ctx_k[c0:c1]]))
        fv.append(np.concatenate([ins.v[i0:i1], kv.ctx_v[c0:c1]]))
        fq.append(np.concatenate([iq[i0:i1], pq.ctx_q[c0:c1]]))
        flen.append(len(fk[-1]))
    db = DecodeBatch(flen, st.q_count.tolist(), wl.hq, wl.hkv, wl.head_dim, wl.dtype,
                     max(8, int(st.seg_len0.max())), rope_base=wl.rope_base)
    db.load_context(0, np.concatenate(fk), np.concatenate(fv))
    db.load_segments(0, kv.seg_k, kv.seg_v, st.seg_len0)
    q_ctx, q_seg = db.pack_prefill_queries(np.concatenate(fq), pq.seg_q, st.seg_len0)
    oc, os_ = db.prefill_outputs()
    bound = max(int(st.seg_len0[st.q_start[b]:st.q_start[b + 1]].sum()) for b in range(wl.num_prompts))
    stream = torch.cuda.current_stream()
    for _ in range(warmup):
        db.prefill(0, q_ctx, q_seg, oc, os_, bound)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record(stream)
    for _ in range(reps):
        db.prefill(0, q_ctx, q_seg, oc, os_, bound)
    e1.record(stream)
    torch.cuda.synchronize()
    assert db.err_flag() == 0
    return e0.elapsed_time(e1) / 1e3 / reps


def run(name: str, reps: int, warmup: int, tile_rows: int = 0):
    import torch
    from paper_2609_05707_amd.session import DecodeBatch

    wl = make(name)
    st = W.make_structure(wl)
    kv = W.layer_kv(st)
    pq = W.prefill_queries(st)
    cap = max(8, int(st.seg_len0.max()))
    ins = iq = None
    extra = {}
    if "instr" in WORKLOADS[name]:
        cpi, lp = WORKLOADS[name]["instr"]
        ins = W.instructions(st, cpi, lp)
        iq = W.instruction_queries(st, ins)
        extra = dict(instr_len=ins.lp.tolist(), instr_prompt_start=ins.prompt_start.tolist())
    db = DecodeBatch(st.ctx_len.tolist(), st.q_count.tolist(), wl.hq, wl.hkv, wl.head_dim, wl.dtype, cap,
                     rope_base=wl.rope_base, tile_rows=tile_rows, **extra)
    if ins is not None:
        db.load_instructions(0, ins.k, ins.v)
    db.load_context(0, kv.ctx_k, kv.ctx_v)
    db.load_segments(0, kv.seg_k, kv.seg_v, st.seg_len0)
    q_ctx, q_seg = db.pack_prefill_queries(pq.ctx_q, pq.seg_q, st.seg_len0, instr_q=iq)
    oc, os_ = db.prefill_outputs()
    bound = max(int(st.seg_len0[st.q_start[b]:st.q_start[b + 1]].sum()) for b in range(wl.num_prompts))
    stream = torch.cuda.current_stream()

    def timed(standard):
        for _ in range(warmup):
            db.prefill(0, q_ctx, q_seg, oc, os_, bound, standard=standard)
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        for _ in range(reps):
            db.prefill(0, q_ctx, q_seg, oc, os_, bound, standard=standard)
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / 1e3 / reps

    # clocks ramp over the first tens of milliseconds of work: without this the
    # path timed first came out ~9% slow even after 30 warmup calls
    t0 = time.perf_counter()
    while time.perf_counter() - t0 < 0.2:
        for _ in range(4):
            db.prefill(0, q_ctx, q_seg, oc, os_, bound)
        torch.cuda.synchronize()
    t_ippd = timed(False)
    t_std = timed(True)
    assert db.err_flag() == 0
    folded = None
    if ins is not None:
        folded = folded_time(st, kv, pq, ins, iq, reps, warmup)
    tokens = int(st.ctx_start[-1] + st.seg_start[-1]) + (0 if ins is None else int(ins.tok_start[-1]))
    f_ippd, f_std = flops(st, False, ins), flops(st, True, ins)
    achieved = f_ippd / t_ippd / 1e12
    res = {
        "metric": "stacked-prompt prefill attention: header tokens/s, 1 MI355X",
        "value": round(tokens / t_ippd, 1),
        "unit": "header tokens/s",
        "n_gpus": 1,
        "reps": reps,
        "warmup": warmup,
        "ms_per_call": round(t_ippd * 1e3, 4),
        "higher_is_better": True,
        "dtype": "bf16",
        "data": "synthetic (seeded normal K/V/Q, rounded to bf16; no dataset)",
        "config": {"workload": f"{name}: B={wl.num_prompts}, Hq={wl.hq}, Hkv={wl.hkv}, D={wl.head_dim}, "
                               f"Lc={wl.ctx_len}, N={wl.questions}, question tokens "
                               f"{wl.question_tokens or wl.seg_len}"
                               + ("" if ins is None else f", {len(ins.lp)} instructions of {ins.lp.tolist()} tokens"),
                   "header_tokens": tokens, "layers": 1},
        "roofline": {"bound": "mfma", "kernel": "prefill_kernel (one ippd_prefill_attention call)",
                     "achieved": round(achieved, 1), "peak": MFMA_BF16_PEAK_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(achieved / MFMA_BF16_PEAK_TFLOPS, 4), "traffic": None,
                     "algorithmic_flops_per_call": f_ippd, "avg_call_us": round(t_ippd * 1e6, 2)},
        "standard": {"ms_per_call": round(t_std * 1e3, 4), "algorithmic_flops_per_call": f_std,
                     "achieved_tflops": round(f_std / t_std / 1e12, 1), "ippd_speedup": round(t_std / t_ippd, 3),
                     "flop_ratio": round(f_std / f_ippd, 3)},
    }
    if folded is not None:
        res["folded_one_level"] = {
            "ms_per_call": round(folded * 1e3, 4), "two_level_speedup": round(folded / t_ippd, 3),
            "note": "the same prompts as a one-level batch whose contexts each carry their own copy of "
                    "the instruction (IPPD prefill): the instruction rows and tiles once per context"}
    return res


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--workload", default="all", choices=["all", *WORKLOADS])
    ap.add_argument("--reps", type=int, default=30)
    ap.add_argument("--warmup", type=int, default=30, help="untimed calls first (a few leave clocks ramping)")
    ap.add_argument("--sweep", choices=["questions", "context"], default=None)
    ap.add_argument("--tile-rows", type=int, default=0, help="rows per unit: 128 or 256 (0 = the planner's choice)")
    args = ap.parse_args()
    import torch
    assert torch.cuda.is_available(), "bench_prefill.py needs a GPU"
    torch.cuda.set_device(0)
    if args.sweep:
        rows = []
        for name, n, lc in sweep_points(args.sweep):
            r = run(name, args.reps, args.warmup, args.tile_rows)
            print(json.dumps(r), flush=True)
            rows.append((n, lc, r["ms_per_call"], r["standard"]["ms_per_call"], r["standard"]["ippd_speedup"],
                         r["standard"]["flop_ratio"], r["roofline"]["achieved"]))
        print("| N | Lc | IPPD ms | standard ms | speedup | FLOP ratio | IPPD TFLOP/s |")
        print("|---|---|---|---|---|---|---|")
        for n, lc, a, b, sp, fr, tf in rows:
            print(f"| {n} | {lc} | {a:.3f} | {b:.3f} | {sp:.2f} | {fr:.2f} | {tf:.0f} |")
        return
    names = list(WORKLOADS) if args.workload == "all" else [args.workload]
    for n in names:
        print(json.dumps(run(n, args.reps, args.warmup, args.tile_rows)), flush=True)


if __name__ == "__main__":
    main()
