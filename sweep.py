#!/usr/bin/env python3
"""Kernel-level analogue of the paper's ablations on one MI355X.

The paper varies the number of questions that share a context (1 to 32,
App. D, questions-per-context ablation) and the context length (1x to 8x,
App. D, context-length ablation) and reports where IPPD gains over standard
decoding.  This script does the same for the decode-step attention alone:
for each point it builds a synthetic Llama-3-8B-shaped batch (one prompt,
Hq 32, Hkv 8, D 128, bf16, question 32 tokens + U{0..64} fed answer tokens,
values N(0,1)*0.5), captures S decode steps x L emulated layers of the fused
IPPD step and of the standard step (the context re-read once per question)
into HIP graphs, replays them on identical KV and reports microseconds per
layer-step, effective tokens/s and the measured speedup next to the
algorithmic byte ratio.  L layers with distinct buffers keep each
layer-step's reads in HBM rather than in the 256 MB Infinity Cache.

Usage: python sweep.py [--kind questions|context|both] [--steps 16]
           [--replays 3] [--out results.jsonl]
One JSON line per point on stdout (and in --out), then a markdown table.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

import workload as W  # noqa: E402
from bench import step_bytes  # noqa: E402

QUESTION_POINTS = [1, 2, 4, 8, 16, 32]          # at Lc 4096
CONTEXT_POINTS = [2048, 4096, 8192, 16384]       # 1x .. 8x of 2048, at N 16


def point_workload(n: int, lc: int, steps: int) -> W.DecodeWorkload:
    return W.custom_workload(wid=300 + n + lc // 512, name=f"sweep-n{n}-lc{lc}", dtype="bf16", num_prompts=1,
                             hq=32, hkv=8, head_dim=128, ctx_len=(lc, lc), questions=(n, n),
                             question_tokens=32, seg_len=(0, 64), steps=steps, value_std=0.5)


def measure(n: int, lc: int, steps: int, replays: int):
    import torch
    from paper_2609_05707_amd.driver import DecodeLoop
    from paper_2609_05707_amd.session import DecodeBatch

    wl = point_workload(n, lc, steps)
    st = W.make_structure(wl)
    ib = float(np.mean([step_bytes(st, t) for t in range(steps)]))
    sb = float(np.mean([step_bytes(st, t, standard=True) for t in range(steps)]))
    layers = int(min(32, max(1, math.ceil((512 << 20) / ib))))
    cap = int(st.seg_len0.max()) + steps + 8
    db = DecodeBatch(st.ctx_len.tolist(), st.q_count.tolist(), wl.hq, wl.hkv, wl.head_dim, wl.dtype, cap,
                     rope_base=wl.rope_base, layers=layers)
    kv = W.layer_kv(st, 0)
    db.load_context(0, kv.ctx_k, kv.ctx_v)
    db.load_segments(0, kv.seg_k, kv.seg_v, st.seg_len0)
    for l in range(1, layers):
        db.ctx_k[l].copy_(db.ctx_k[0]); db.ctx_vt[l].copy_(db.ctx_vt[0])
        db.seg_k[l].copy_(db.seg_k[0]); db.seg_vt[l].copy_(db.seg_vt[0])
        db.seg_len[l].copy_(db.seg_len[0])
    q, k, v, act = [], [], [], []
    for t in range(steps):
        si = W.step_inputs(st, t)
        q.append(db.to_dev(si.q_new)); k.append(db.to_dev(si.k_new)); v.append(db.to_dev(si.v_new))
        act.append(torch.from_numpy(si.active.astype(np.uint8)).to(db.device))
    res = {}
    for name, standard in (("ippd", False), ("standard", True)):
        loop = DecodeLoop(db, q, k, v, act, standard=standard)
        loop.capture()
        loop.replay()                               # warm-up
        torch.cuda.synchronize()
        times = []
        for _ in range(replays):
            loop.reset()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record()
            loop.replay()
            e1.record()
            torch.cuda.synchronize()
            times.append(e0.elapsed_time(e1) / 1e3)
        res[name] = min(times) / (steps * layers)
        loop.reset()
        assert db.err_flag() == 0
    tokens = float(np.mean([st.active(t).sum() for t in range(steps)]))
    return {
        "questions": n, "ctx_len": lc, "layers_cycled": layers, "steps": steps,
        "ippd_us_per_layer_step": round(res["ippd"] * 1e6, 3),
        "standard_us_per_layer_step": round(res["standard"] * 1e6, 3),
        "ippd_tokens_per_s": round(tokens / res["ippd"], 1),
        "standard_tokens_per_s": round(tokens / res["standard"], 1),
        "speedup": round(res["standard"] / res["ippd"], 3),
        "algorithmic_byte_ratio": round(sb / ib, 3),
        "ippd_hbm_gbps": round(ib / res["ippd"] / 1e9, 1),
        "standard_hbm_gbps": round(sb / res["standard"] / 1e9, 1),
    }


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--kind", choices=["questions", "context", "both"], default="both")
    ap.add_argument("--steps", type=int, default=16)
    ap.add_argument("--replays", type=int, default=3)
    ap.add_argument("--out", default=None)
    args = ap.parse_args()
    import torch
    assert torch.cuda.is_available(), "sweep.py needs a GPU"
    torch.cuda.set_device(0)
    points = []
    if args.kind in ("questions", "both"):
        points += [(n, 4096) for n in QUESTION_POINTS]
    if args.kind in ("context", "both"):
        points += [(16, lc) for lc in CONTEXT_POINTS if (16, lc) not in points]
    rows = []
    out = open(args.out, "w") if args.out else None
    for n, lc in points:
        r = measure(n, lc, args.steps, args.replays)
        rows.append(r)
        line = json.dumps(r)
        print(line, flush=True)
        if out:
            out.write(line + "\n")
            out.flush()
    print("\n| N | Lc | IPPD us/layer-step | standard us/layer-step | speedup | byte ratio | IPPD GB/s |")
    print("|---|---|---|---|---|---|---|")
    for r in rows:
        print(f"| {r['questions']} | {r['ctx_len']} | {r['ippd_us_per_layer_step']} | "
              f"{r['standard_us_per_layer_step']} | {r['speedup']} | {r['algorithmic_byte_ratio']} | "
              f"{r['ippd_hbm_gbps']} |")


if __name__ == "__main__":
    main()
