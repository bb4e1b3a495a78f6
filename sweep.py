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
CPI_POINTS = [1, 2, 4, 6]                        # contexts per instruction (two-level sharing)
TWO_LEVEL = dict(contexts=12, instr=2048, ctx=1024, questions=8)


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


def _replay_us(loop, steps, layers, replays):
    import torch
    loop.capture()
    loop.replay()
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
    loop.reset()
    return min(times) / (steps * layers) * 1e6


def measure_two_level(cpi: int, steps: int, replays: int):
    """Contexts per instruction (Sec. 4.4, C/P): 12 contexts of 1024 tokens with 8
    questions each behind instructions of 2048 tokens, cpi contexts per
    instruction.  Three layouts on identical values: two-level (p read once per
    instruction), folded (every context carries its own copy of p) and the
    standard baseline on the folded layout (p + c read per question)."""
    import torch
    from paper_2609_05707_amd.driver import DecodeLoop
    from paper_2609_05707_amd.session import DecodeBatch

    cfg = TWO_LEVEL
    wl = W.custom_workload(wid=700 + cpi, name=f"two-level-cpi{cpi}", dtype="bf16", num_prompts=cfg["contexts"],
                           hq=32, hkv=8, head_dim=128, ctx_len=(cfg["ctx"], cfg["ctx"]),
                           questions=(cfg["questions"], cfg["questions"]), question_tokens=12, seg_len=(0, 28),
                           steps=steps, value_std=0.5)
    st = W.make_structure(wl)
    ins = W.instructions(st, cpi, (cfg["instr"], cfg["instr"]))
    kv = W.layer_kv(st)
    e = 2
    per_tok = 2 * wl.hkv * wl.head_dim * e
    tail = sum(int(st.active(t).sum()) for t in range(steps)) / steps * (
        (wl.hq + 4 * wl.hkv) * wl.head_dim * e + wl.hq * wl.head_dim * 4)
    seg = float(np.mean([np.sum(st.seg_len_at(t)[st.active(t)]) for t in range(steps)])) * per_tok
    nt, S = st.num_questions, len(ins.lp)
    bytes_two = S * cfg["instr"] * per_tok + cfg["contexts"] * cfg["ctx"] * per_tok + seg + tail
    bytes_fold = cfg["contexts"] * (cfg["instr"] + cfg["ctx"]) * per_tok + seg + tail
    bytes_std = nt * (cfg["instr"] + cfg["ctx"]) * per_tok + seg + tail
    layers = int(min(32, max(1, math.ceil((512 << 20) / bytes_two))))
    cap = int(st.seg_len0.max()) + steps + 8

    def inputs(db):
        q, k, v, act = [], [], [], []
        for t in range(steps):
            si = W.step_inputs(st, t)
            q.append(db.to_dev(si.q_new)); k.append(db.to_dev(si.k_new)); v.append(db.to_dev(si.v_new))
            act.append(torch.from_numpy(si.active.astype(np.uint8)).to(db.device))
        return q, k, v, act

    def replicate(db):
        for l in range(1, layers):
            db.ctx_k[l].copy_(db.ctx_k[0]); db.ctx_vt[l].copy_(db.ctx_vt[0])
            db.seg_k[l].copy_(db.seg_k[0]); db.seg_vt[l].copy_(db.seg_vt[0])
            db.seg_len[l].copy_(db.seg_len[0])

    # two-level
    db2 = DecodeBatch(st.ctx_len.tolist(), st.q_count.tolist(), wl.hq, wl.hkv, wl.head_dim, wl.dtype, cap,
                      rope_base=wl.rope_base, layers=layers, instr_len=ins.lp.tolist(),
                      instr_prompt_start=ins.prompt_start.tolist())
    db2.load_instructions(0, ins.k, ins.v)
    db2.load_context(0, kv.ctx_k, kv.ctx_v)
    db2.load_segments(0, kv.seg_k, kv.seg_v, st.seg_len0)
    replicate(db2)
    t_two = _replay_us(DecodeLoop(db2, *inputs(db2)), steps, layers, replays)
    assert db2.err_flag() == 0
    del db2
    # folded: context b := [p_s(b); c_b]
    s_of = np.searchsorted(ins.prompt_start, np.arange(wl.num_prompts), side="right") - 1
    fk = np.concatenate([np.concatenate([ins.k[ins.tok_start[s_of[b]]:ins.tok_start[s_of[b] + 1]],
                                         kv.ctx_k[st.ctx_start[b]:st.ctx_start[b + 1]]]) for b in range(wl.num_prompts)])
    fv = np.concatenate([np.concatenate([ins.v[ins.tok_start[s_of[b]]:ins.tok_start[s_of[b] + 1]],
                                         kv.ctx_v[st.ctx_start[b]:st.ctx_start[b + 1]]]) for b in range(wl.num_prompts)])
    flen = [cfg["instr"] + cfg["ctx"]] * wl.num_prompts
    db1 = DecodeBatch(flen, st.q_count.tolist(), wl.hq, wl.hkv, wl.head_dim, wl.dtype, cap,
                      rope_base=wl.rope_base, layers=layers)
    db1.load_context(0, fk, fv)
    db1.load_segments(0, kv.seg_k, kv.seg_v, st.seg_len0)
    replicate(db1)
    q = inputs(db1)
    t_fold = _replay_us(DecodeLoop(db1, *q), steps, layers, replays)
    t_std = _replay_us(DecodeLoop(db1, *q, standard=True), steps, layers, replays)
    assert db1.err_flag() == 0
    tokens = float(np.mean([st.active(t).sum() for t in range(steps)]))
    return {
        "contexts_per_instruction": cpi, "instructions": S, "contexts": cfg["contexts"], "instr_len": cfg["instr"],
        "ctx_len": cfg["ctx"], "questions_per_context": cfg["questions"], "layers_cycled": layers, "steps": steps,
        "two_level_us_per_layer_step": round(t_two, 3), "folded_us_per_layer_step": round(t_fold, 3),
        "standard_us_per_layer_step": round(t_std, 3),
        "two_level_tokens_per_s": round(tokens / t_two * 1e6, 1),
        "speedup_vs_folded": round(t_fold / t_two, 3), "speedup_vs_standard": round(t_std / t_two, 3),
        "byte_ratio_folded": round(bytes_fold / bytes_two, 3), "byte_ratio_standard": round(bytes_std / bytes_two, 3),
        "two_level_hbm_gbps": round(bytes_two / t_two / 1e3, 1),
    }


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--kind", choices=["questions", "context", "both", "two-level", "all"], default="both")
    ap.add_argument("--steps", type=int, default=16)
    ap.add_argument("--replays", type=int, default=3)
    ap.add_argument("--out", default=None)
    args = ap.parse_args()
    import torch
    assert torch.cuda.is_available(), "sweep.py needs a GPU"
    torch.cuda.set_device(0)
    points = []
    if args.kind in ("questions", "both", "all"):
        points += [(n, 4096) for n in QUESTION_POINTS]
    if args.kind in ("context", "both", "all"):
        points += [(16, lc) for lc in CONTEXT_POINTS if (16, lc) not in points]
    rows = []
    out = open(args.out, "w") if args.out else None
    if args.kind in ("two-level", "all"):
        tl = []
        for cpi in CPI_POINTS:
            r = measure_two_level(cpi, args.steps, args.replays)
            tl.append(r)
            print(json.dumps(r), flush=True)
            if out:
                out.write(json.dumps(r) + "\n")
                out.flush()
        print("\n| contexts per instruction | two-level us | folded us | standard us | vs folded | vs standard "
              "| byte ratio folded | byte ratio standard |")
        print("|---|---|---|---|---|---|---|---|")
        for r in tl:
            print(f"| {r['contexts_per_instruction']} | {r['two_level_us_per_layer_step']} | "
                  f"{r['folded_us_per_layer_step']} | {r['standard_us_per_layer_step']} | {r['speedup_vs_folded']} | "
                  f"{r['speedup_vs_standard']} | {r['byte_ratio_folded']} | {r['byte_ratio_standard']} |")
    for n, lc in points:
        r = measure(n, lc, args.steps, args.replays)
        rows.append(r)
        line = json.dumps(r)
        print(line, flush=True)
        if out:
            out.write(line + "\n")
            out.flush()
    if not rows:
        return
    print("\n| N | Lc | IPPD us/layer-step | standard us/layer-step | speedup | byte ratio | IPPD GB/s |")
    print("|---|---|---|---|---|---|---|")
    for r in rows:
        print(f"| {r['questions']} | {r['ctx_len']} | {r['ippd_us_per_layer_step']} | "
              f"{r['standard_us_per_layer_step']} | {r['speedup']} | {r['algorithmic_byte_ratio']} | "
              f"{r['ippd_hbm_gbps']} |")


if __name__ == "__main__":
    main()
