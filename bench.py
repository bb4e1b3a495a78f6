#!/usr/bin/env python3
"""Benchmark of the IPPD decode-step hot path on one MI355X.

A step is one decode step of the workload: for every emulated layer, one
ippd_decode_step call (virtual-position rotation + KV append, shared-context
and own-segment attention, exact merge; two kernel launches), queued
back-to-back on one stream with all inputs resident in HBM.  Each layer has
its own KV cache (same values, distinct buffers), so a step streams every
layer's context from HBM rather than from the 256 MB Infinity Cache.

value = effective decode tokens/s = sum over timed steps and layers of the
active questions, divided by the wall time of the timed steps (a
layer-level figure: each layer-step decodes one token per active question
at that layer).  The same steps are then re-run with the standard baseline
(standard_decode_step, the context re-read once per question) on
identical KV, and the fp64 oracle is timed on a bounded sample on the host.
Beside the headline: the separate-call and graph-replay timings, the warm
figure (one layer buffer cycled) and single calls timed after a 512 MiB
cache scrub.
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

HBM_PEAK_GBPS = 8000.0
MFMA_BF16_PEAK_TFLOPS = 2500.0
METRIC = "effective decode tokens/s (questions×steps/s) + HBM GB/s % of peak, 1 MI355X"

DEFAULT_LAYERS = {1: 1, 2: 32, 3: 1, 4: 4, 5: 32}


def parse():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=None, help="timed decode steps (default: the workload's)")
    ap.add_argument("--warmup", type=int, default=8)
    ap.add_argument("--workload", type=int, default=5,
                    help="workload id (1..5); 5, the largest one-GPU workload, is the headline")
    ap.add_argument("--layers", type=int, default=None, help="emulated layers cycled per step")
    ap.add_argument("--no-standard", action="store_true", help="skip the standard baseline")
    ap.add_argument("--no-cpu-baseline", action="store_true", help="skip the oracle timing")
    ap.add_argument("--no-dense", action="store_true", help="skip the dense-mask baseline")
    ap.add_argument("--no-warm", action="store_true",
                    help="skip the warm single-buffer and scrubbed single-call timings (every call cold)")
    ap.add_argument("--cpu-sample", type=int, default=None,
                    help="question-steps the oracle computes (default: 400, 240 on the 32-layer workload)")
    ap.add_argument("--chunk", type=int, default=0, help="context tokens per unit (0 = library default)")
    ap.add_argument("--tile-rows", type=int, default=0, help="rows per context unit (0 = library default)")
    ap.add_argument("--standard-only", action="store_true",
                    help="profiling aid: run only the standard baseline's timed steps (no JSON line); its "
                         "kernels are then the only decode kernels a counter run sees")
    return ap.parse_args()


# ----------------------------------------------------------------- accounting

def step_bytes(st: W.Structure, t: int, standard: bool = False) -> int:
    """Algorithmic HBM bytes of one fused layer-step at step t.

    Per prompt with an active question: its context K and V once (IPPD) or once
    per active question (standard), 2*Lc*Hkv*D*e.  Per active question: its cached
    segment K and V (2*s*Hkv*D*e), the raw q/k/v of the fed token
    ((Hq + 2*Hkv)*D*e), the appended key/value (2*Hkv*D*e) and the fp32 output
    rows (Hq*D*4 + Hq*4 for lse)."""
    wl = st.wl
    e = wl.elem_bytes
    D, hq, hkv = wl.head_dim, wl.hq, wl.hkv
    act = st.active(t)
    seg = st.seg_len_at(t)
    tot = 0
    for b in range(wl.num_prompts):
        q0, q1 = st.q_start[b], st.q_start[b + 1]
        n_act = int(act[q0:q1].sum())
        if n_act == 0:
            continue
        ctx = 2 * int(st.ctx_len[b]) * hkv * D * e
        tot += ctx * (n_act if standard else 1)
    ia = np.flatnonzero(act)
    tot += int(np.sum(2 * seg[ia] * hkv * D * e))
    tot += len(ia) * ((hq + 2 * hkv) * D * e + 2 * hkv * D * e + hq * D * 4 + hq * 4)
    return tot


def step_flops(st: W.Structure, t: int) -> int:
    wl = st.wl
    act = st.active(t)
    seg = st.seg_len_at(t)
    tot = 0
    for i in np.flatnonzero(act):
        b = st.prompt_of[i]
        tot += 4 * wl.hq * wl.head_dim * (int(st.ctx_len[b]) + int(seg[i]) + 1)
    return tot


def dense_flops(st: W.Structure, t: int) -> int:
    """FLOPs of the dense-mask form: the context part as IPPD, the segment part
    every active row of a prompt against the segments of all its questions."""
    wl = st.wl
    act = st.active(t)
    seg = st.seg_len_at(t) + act                  # the step's token is appended first
    tot = 0
    for b in range(wl.num_prompts):
        q0, q1 = st.q_start[b], st.q_start[b + 1]
        n_act = int(act[q0:q1].sum())
        tot += 4 * wl.hq * wl.head_dim * n_act * (int(st.ctx_len[b]) + int(seg[q0:q1].sum()))
    return tot


def read_traffic(workload_id: int, path_kind: str = "decode"):
    """HBM traffic per attention launch from the committed rocprofv3 counter summary
    (path_kind "decode": the IPPD step, "standard": the standard baseline's step),
    only if it was taken on the current kernel sources."""
    path = os.path.join(ROOT, "profiles", f"traffic_{path_kind}_step_wl{workload_id}.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    from paper_2609_05707_amd.traffic import kernel_source_hash
    if rec.get("kernel_source_hash") != kernel_source_hash():
        return None
    return rec.get("hbm_bytes_per_launch")


# ----------------------------------------------------------------- cpu oracle

def cpu_baseline(st: W.Structure, kv: W.LayerKV, n_samples: int):
    """Time the fp64 oracle on the first question-steps of the workload (layer 0)
    with the BLAS threads it finds, and on the tiny fp32 workload also with one."""
    try:
        from threadpoolctl import threadpool_info, threadpool_limits
        threads = max([p.get("num_threads", 1) for p in threadpool_info()] or [1])
    except Exception:
        threadpool_limits = None
        threads = 1
    rec = _oracle_timing(st, kv, n_samples)
    rec.update({"cores": int(threads), "host_cpus": os.cpu_count()})
    if st.wl.wid == 1 and threadpool_limits is not None:
        with threadpool_limits(limits=1):
            one = _oracle_timing(st, kv, n_samples)
        rec["one_thread"] = {"value": one["value"], "unit": "tokens/s", "cores": 1, "seconds": one["seconds"]}
    return rec


def sample_steps(wl: W.DecodeWorkload):
    """Steps at which the oracle sample is taken: the first steps, except on the
    32-layer workload, whose active set shrinks over 128 steps: there the steps
    0, 15, 64 and the last, so that the sample spans the shrinking set."""
    if wl.wid == 5:
        return [0, 15, 64, wl.steps - 1]
    return list(range(wl.steps))


def _oracle_timing(st: W.Structure, kv: W.LayerKV, n_samples: int):
    from oracle import ippd as O
    state = O.KVState.from_packed(kv.seg_k, kv.seg_v, st.seg_start)
    at = sample_steps(st.wl)
    spread = len(at) < st.wl.steps
    per_step = (n_samples + len(at) - 1) // len(at) if spread else n_samples
    done = 0
    t_total = 0.0
    used = []
    for t in range(st.wl.steps):
        si = W.step_inputs(st, t)
        act = np.flatnonzero(si.active)
        want = min(per_step, n_samples - done) if t in at else 0
        take = act[: max(0, want)]
        if len(take):
            t0 = time.perf_counter()
            O.decode_step_standard(kv.ctx_k, kv.ctx_v, st.ctx_start, st.q_start, state,
                                   si.q_new, si.k_new, si.v_new, si.active, st.wl.rope_base,
                                   questions=take.tolist())
            t_total += time.perf_counter() - t0
            done += len(take)
            used.append(t)
        state.append(si.k_new, si.v_new, si.active)
        if done >= n_samples:
            break
    where = (f"steps {', '.join(str(u) for u in used)}, up to {per_step} active questions each" if spread
             else f"steps 0..{used[-1] if used else 0}")
    return {"value": done / t_total, "unit": "tokens/s", "kind": "oracle",
            "sample": f"{done} question-steps of layer 0 ({where}; all heads), "
                      f"{t_total:.1f} s of fp64 numpy",
            "seconds": round(t_total, 2)}


# ----------------------------------------------------------------------- main

def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (asked for --gpus {args.gpus}); the decode-attention "
              "path runs on a single MI355X; sharding over several GPUs is not implemented.",
              file=sys.stderr)
        sys.exit(2)
    import torch
    from paper_2609_05707_amd.session import DecodeBatch

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    wl = W.workload(args.workload)
    st = W.make_structure(wl)
    steps = args.steps if args.steps is not None else wl.steps
    layers = args.layers if args.layers is not None else DEFAULT_LAYERS[wl.wid]
    data_steps = wl.steps                      # distinct step inputs; cycled if steps > data_steps
    cap = int(st.seg_len0.max()) + max(steps, args.warmup, data_steps) + 8
    db = DecodeBatch(st.ctx_len.tolist(), st.q_count.tolist(), wl.hq, wl.hkv, wl.head_dim, wl.dtype,
                     cap, rope_base=wl.rope_base, layers=layers, chunk_tokens=args.chunk,
                     tile_rows=args.tile_rows)
    kv0 = W.layer_kv(st, 0)
    db.load_context(0, kv0.ctx_k, kv0.ctx_v)
    db.load_segments(0, kv0.seg_k, kv0.seg_v, st.seg_len0)
    for l in range(1, layers):
        db.ctx_k[l].copy_(db.ctx_k[0]); db.ctx_vt[l].copy_(db.ctx_vt[0])
        db.seg_k[l].copy_(db.seg_k[0]); db.seg_vt[l].copy_(db.seg_vt[0])
        db.seg_len[l].copy_(db.seg_len[0])
    seg0 = db.seg_len[0].clone()
    nt = st.num_questions
    # per-step inputs resident on the device
    qs, ks, vs, acts = [], [], [], []
    for t in range(data_steps):
        si = W.step_inputs(st, t)
        qs.append(db.to_dev(si.q_new)); ks.append(db.to_dev(si.k_new)); vs.append(db.to_dev(si.v_new))
        acts.append(torch.from_numpy(si.active.astype(np.uint8)).to(db.device))
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()

    def set_step_active(t, nl=None):
        ptr = acts[t % data_steps].data_ptr()
        for bt in db.batches[: layers if nl is None else nl]:
            bt.active = ptr

    def reset():
        for l in range(layers):
            db.seg_len[l].copy_(seg0)
        torch.cuda.synchronize()

    def run(n_steps, standard=False, events=None, separate=False, dense=False, nl=None):
        for t in range(n_steps):
            d = t % data_steps
            set_step_active(d, nl)
            for l in range(layers if nl is None else nl):
                if events is not None:
                    events[t][l][0].record(stream)
                if separate or dense:
                    db.append(l, qs[d], ks[d], vs[d])
                    db.decode(l, standard=standard, dense=dense)
                else:
                    db.decode_step(l, qs[d], ks[d], vs[d], standard=standard, write_q_rot=False)
                if events is not None:
                    events[t][l][1].record(stream)

    def timed(standard=False, separate=False, dense=False, nl=None):
        reset()
        run(args.warmup, standard, separate=separate, dense=dense, nl=nl)
        reset()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(stream)
        run(steps, standard, separate=separate, dense=dense, nl=nl)
        e1.record(stream)
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / 1e3

    def scrubbed_call_time():
        """Cross-check of the cold figure: layer 0 only, one decode-step call per
        step timed alone (HIP events around it), after a 512 MiB write that
        evicts the caches (L2 and the 256 MB Infinity Cache)."""
        scrub = torch.empty(512 << 20, dtype=torch.uint8, device=db.device)
        reset()
        durs = []
        for t in range(steps):
            d = t % data_steps
            set_step_active(d, 1)
            scrub.fill_(t & 0xFF)
            a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            a.record(stream)
            db.decode_step(0, qs[d], ks[d], vs[d], write_q_rot=False)
            b.record(stream)
            torch.cuda.synchronize()
            durs.append(a.elapsed_time(b) / 1e3)
        del scrub
        reset()
        return float(np.mean(durs))

    def kernel_time(standard=False):
        """Average duration of one decode-step call (its two launches), from HIP events
        around each call on the launching stream, over a second pass of the same steps."""
        reset()
        run(args.warmup, standard)
        reset()
        ev = [[(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
               for _ in range(layers)] for _ in range(steps)]
        torch.cuda.synchronize()
        run(steps, standard, events=ev)
        torch.cuda.synchronize()
        durs = [a.elapsed_time(b) / 1e3 for row in ev for (a, b) in row]
        return float(np.mean(durs)), durs

    if args.standard_only:
        t_std = timed(True)
        print(f"standard only: {t_std / (steps * layers) * 1e6:.3f} us per layer-step, err flag {db.err_flag()}",
              file=sys.stderr)
        return
    t_ippd = timed(False)
    err = db.err_flag()
    tokens = sum(int(st.active(t % data_steps).sum()) for t in range(steps)) * layers
    value = tokens / t_ippd
    step_b = [step_bytes(st, t % data_steps) for t in range(steps)]
    bytes_total = sum(step_b) * layers
    flops_total = sum(step_flops(st, t % data_steps) for t in range(steps)) * layers
    k_avg, k_durs = kernel_time(False)
    # average call time per quarter of the steps (the active set shrinks over them)
    quarters = np.array_split(np.asarray(k_durs).reshape(steps, layers), min(4, steps))
    k_quarters = [round(float(np.mean(qq)) * 1e6, 3) for qq in quarters]
    bytes_per_launch = float(np.mean(step_b))
    achieved = bytes_per_launch / k_avg / 1e9
    traffic = read_traffic(wl.wid)
    t_sep = timed(False, separate=True)
    flags = {"ippd": err, "separate": db.err_flag()}

    def graph_time(nl=None):
        """The same steps captured once into a HIP graph and replayed (kernels and
        arguments of the eager sequence; no host launch cost in the timed region),
        over all layer buffers or the first nl."""
        from paper_2609_05707_amd.driver import DecodeLoop
        reset()                                   # the loop restores the lengths it starts from
        loop = DecodeLoop(db, [qs[t % data_steps] for t in range(steps)], [ks[t % data_steps] for t in range(steps)],
                          [vs[t % data_steps] for t in range(steps)], [acts[t % data_steps] for t in range(steps)],
                          layers=nl)
        loop.capture()
        loop.replay()
        torch.cuda.synchronize()
        best = None
        for _ in range(3):
            loop.reset()
            torch.cuda.synchronize()
            e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
            e0.record(stream)
            loop.replay()
            e1.record(stream)
            torch.cuda.synchronize()
            dt = e0.elapsed_time(e1) / 1e3
            best = dt if best is None else min(best, dt)
        loop.reset()
        return best

    t_graph = graph_time()
    flags["graph"] = db.err_flag()
    # the same steps on one layer buffer only (warm: the step's bytes may stay in
    # the Infinity Cache between steps; replayed from a graph, since one call per
    # step leaves the host's launch cost exposed), and single calls after a cache scrub
    t_warm = t_scrub = None
    if not args.no_warm:
        t_warm = graph_time(nl=1)
        flags["warm"] = db.err_flag()
        t_scrub = scrubbed_call_time()
        flags["scrubbed"] = db.err_flag()

    result = {
        "metric": METRIC,
        "value": round(value, 1),
        "unit": "tokens/s",
        "n_gpus": 1,
        "steps": steps,
        "warmup": args.warmup,
        "ms_per_step": round(t_ippd / steps * 1e3, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16" if wl.dtype == "bf16" else "f32",
        "data": "synthetic (seeded normal K/V/Q, rounded to bf16; no dataset)",
        "config": {
            "workload": f"{wl.name}: B={wl.num_prompts}, Hq={wl.hq}, Hkv={wl.hkv}, D={wl.head_dim}, "
                        f"Lc={wl.ctx_len}, N={wl.questions}, {wl.steps} decode steps",
            "layers_cycled": layers,
            "chunk_tokens": args.chunk or "auto",
            "tile_rows": args.tile_rows or "auto",
            "step": "per layer: one ippd_decode_step call (append + attention + merge, two launches)",
            "us_per_layer_step": round(t_ippd / (steps * layers) * 1e6, 3),
            "separate_calls_us_per_layer_step": round(t_sep / (steps * layers) * 1e6, 3),
            "graph_replay_us_per_layer_step": round(t_graph / (steps * layers) * 1e6, 3),
            "warm_single_buffer_graph_us_per_layer_step": None if t_warm is None else round(t_warm / steps * 1e6, 3),
            "scrubbed_single_call_us": None if t_scrub is None else round(t_scrub * 1e6, 3),
        },
        "hbm_gbps": round(bytes_total / t_ippd / 1e9, 1),
        "hbm_frac": round(bytes_total / t_ippd / 1e9 / HBM_PEAK_GBPS, 4),
        "mfma_tflops": round(flops_total / t_ippd / 1e12, 2),
        "roofline": {
            "bound": "hbm",
            "kernel": "attend_kernel + merge_kernel (one ippd_decode_step call)",
            "achieved": round(achieved, 1),
            "peak": HBM_PEAK_GBPS,
            "unit": "GB/s",
            "frac": round(achieved / HBM_PEAK_GBPS, 4),
            "traffic": traffic,
            "algorithmic_bytes_per_launch": int(bytes_per_launch),
            "avg_launch_us": round(k_avg * 1e6, 3),
            "avg_launch_us_by_step_quarter": k_quarters,
        },
        "err_flag": err,
    }
    if not args.no_standard:
        t_std = timed(True)
        flags["standard"] = db.err_flag()
        std_b = [step_bytes(st, t % data_steps, standard=True) for t in range(steps)]
        ks_avg, _ = kernel_time(True)
        result["standard"] = {
            "value": round(tokens / t_std, 1),
            "ms_per_step": round(t_std / steps * 1e3, 4),
            "ippd_speedup": round(t_std / t_ippd, 3),
            "algorithmic_byte_ratio": round(float(np.mean(std_b)) / bytes_per_launch, 3),
            "avg_launch_us": round(ks_avg * 1e6, 3),
            # per-question context re-reads divided by the call time: an
            # algorithmic-bytes rate (re-reads may be served from L2 or the
            # Infinity Cache), not HBM bandwidth
            "algorithmic_bytes_rate_gbps": round(float(np.mean(std_b)) / ks_avg / 1e9, 1),
            # HBM bytes per call from FETCH_SIZE + WRITE_SIZE counters (null if not taken on these sources)
            "traffic": read_traffic(wl.wid, "standard"),
        }
    if not args.no_dense and db.ws_dense_bytes > 0:
        # the paper's own scheme (dense mask over the whole stacked prompt), as
        # append + attention calls: compare with the IPPD separate calls
        t_dense = timed(False, dense=True)
        flags["dense"] = db.err_flag()
        ippd_f = sum(step_flops(st, t % data_steps) for t in range(steps))
        dense_f = sum(dense_flops(st, t % data_steps) for t in range(steps))
        result["dense_mask"] = {
            "us_per_layer_step": round(t_dense / (steps * layers) * 1e6, 3),
            "vs_ippd_separate_calls": round(t_dense / t_sep, 3),
            "flop_ratio": round(dense_f / ippd_f, 3),
            "note": "append + dense_decode_attention (every row over all keys of its prompt, M_fin mask)",
        }
    result["err_flags"] = flags
    if not args.no_cpu_baseline:
        n_cpu = args.cpu_sample if args.cpu_sample is not None else (240 if wl.wid == 5 else 400)
        result["cpu_baseline"] = cpu_baseline(st, kv0, n_cpu)
    print(json.dumps(result), flush=True)


if __name__ == "__main__":
    main()
