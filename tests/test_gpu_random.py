"""GPU: seeded random configurations against the fp64 oracle.

Each case draws its own small configuration: dtype, head dimension, query
heads per kv head (1..16), prompts, ragged context / question / segment
lengths (empty ones included), chunk size, rows per unit, an optional
instruction level, and the call (fused step, separate calls, standard
baseline, dense-mask baseline; IPPD or standard prefill).  Every configuration is valid by
construction.  Tolerances: 1e-5 for fp32, 2e-2 for bf16."""
import numpy as np
import pytest
import torch

import workload as W
from oracle import ippd as O
from oracle import prefill as P
from paper_2609_05707_amd.session import DecodeBatch
from tests.gpu_harness import log, max_err

pytestmark = pytest.mark.gpu

SENTINEL = -333.0


def tol(dtype):
    return 1e-5 if dtype == "f32" else 2e-2


def draw(k, prefill):
    r = np.random.default_rng([7000 + (500 if prefill else 0), k])
    dtype = str(r.choice(["bf16", "f32"]))
    d = int(r.choice([64, 128]))
    hkv = int(r.choice([1, 2, 4]))
    g = int(r.choice([1, 2, 3, 4, 8, 16]))
    cfg = dict(dtype=dtype, d=d, hkv=hkv, hq=hkv * g, B=int(r.integers(1, 5)),
               ctx=(int(r.integers(0, 40)), int(r.integers(40, 600))),
               qs=(int(r.integers(0, 2)), int(r.integers(2, 8))),
               seg=(int(r.integers(0, 8)), int(r.integers(8, 50))),
               chunk=int(r.choice([0, 32, 96, 256])),
               two_level=bool(r.random() < 0.3), cpi=int(r.integers(1, 4)),
               lp=(int(r.integers(0, 50)), int(r.integers(50, 300))))
    if prefill:
        cfg["rows"] = int(r.choice([0, 128, 256])) if (dtype == "bf16" and d == 128) else 0
        cfg["mode"] = str(r.choice(["ippd", "standard"]))
    else:
        cfg["rows"] = int(r.choice([0, 16, 32, 64, 128] + ([256] if dtype == "bf16" and d == 128 else [])))
        cfg["mode"] = str(r.choice(["fused", "separate", "standard"]))
        # drawn last, so the cases above keep their configurations: the
        # dense-mask baseline on one-level batches
        if r.random() < 0.25 and not cfg["two_level"]:
            cfg["mode"] = "dense"
    return cfg


def make(cfg, wid, steps, question_tokens=0):
    wl = W.custom_workload(wid=wid, dtype=cfg["dtype"], num_prompts=cfg["B"], hq=cfg["hq"], hkv=cfg["hkv"],
                           head_dim=cfg["d"], ctx_len=cfg["ctx"], questions=cfg["qs"],
                           question_tokens=question_tokens, seg_len=cfg["seg"], steps=steps,
                           stop=(1, steps) if steps > 1 else None,
                           value_std=0.5 if cfg["dtype"] == "bf16" else 1.0)
    st = W.make_structure(wl)
    ins = W.instructions(st, cfg["cpi"], cfg["lp"]) if cfg["two_level"] else None
    return wl, st, ins


def batch(st, ins, cfg, cap):
    wl = st.wl
    extra = {} if ins is None else dict(instr_len=ins.lp.tolist(), instr_prompt_start=ins.prompt_start.tolist())
    db = DecodeBatch(st.ctx_len.tolist(), st.q_count.tolist(), wl.hq, wl.hkv, wl.head_dim, wl.dtype, cap,
                     rope_base=wl.rope_base, chunk_tokens=cfg["chunk"], tile_rows=cfg["rows"], **extra)
    kv = W.layer_kv(st)
    if ins is not None:
        db.load_instructions(0, ins.k, ins.v)
    db.load_context(0, kv.ctx_k, kv.ctx_v)
    db.load_segments(0, kv.seg_k, kv.seg_v, st.seg_len0)
    return db, kv


@pytest.mark.parametrize("k", range(24))
def test_random_decode(k):
    cfg = draw(k, prefill=False)
    log(f"case: random decode {k}: {cfg}")
    wl, st, ins = make(cfg, 7000 + k, steps=2)
    db, kv = batch(st, ins, cfg, int(st.seg_len0.max() if st.num_questions else 0) + wl.steps + 8)
    instr = None if ins is None else O.Instructions(ins.prompt_start, ins.tok_start, ins.k, ins.v)
    state = O.KVState.from_packed(kv.seg_k, kv.seg_v, st.seg_start)
    for t in range(wl.steps):
        si = W.step_inputs(st, t)
        db.set_active(si.active)
        q, kk, v = db.to_dev(si.q_new), db.to_dev(si.k_new), db.to_dev(si.v_new)
        db.out.fill_(SENTINEL)
        db.lse.fill_(SENTINEL)
        if cfg["mode"] in ("separate", "dense"):
            db.append(0, q, kk, v)
            db.decode(0, dense=cfg["mode"] == "dense")
        else:
            db.decode_step(0, q, kk, v, standard=cfg["mode"] == "standard")
        torch.cuda.synchronize()
        got = db.out[: st.num_questions].float().cpu().numpy()
        got_lse = db.lse[: st.num_questions].float().cpu().numpy()
        ref, ref_lse = O.decode_step_standard(kv.ctx_k, kv.ctx_v, st.ctx_start, st.q_start, state, si.q_new,
                                              si.k_new, si.v_new, si.active, wl.rope_base, instr=instr)
        state.append(si.k_new, si.v_new, si.active)
        act = si.active
        e = max_err(got[act], ref[act]) if act.any() else 0.0
        el = max_err(got_lse[act], ref_lse[act]) if act.any() else 0.0
        log(f"  step {t}: {int(act.sum())} active, max err out {e:.3e} lse {el:.3e}")
        assert e <= tol(wl.dtype) and el <= tol(wl.dtype)
        assert (got[~act] == SENTINEL).all() and (got_lse[~act] == SENTINEL).all()
    np.testing.assert_array_equal(db.seg_len[0][: st.num_questions].cpu().numpy(), st.seg_len_at(wl.steps))
    assert db.err_flag() == 0


@pytest.mark.parametrize("k", range(12))
def test_random_prefill(k):
    cfg = draw(k, prefill=True)
    log(f"case: random prefill {k}: {cfg}")
    wl, st, ins = make(cfg, 7600 + k, steps=1)
    db, kv = batch(st, ins, cfg, max(8, int(st.seg_len0.max()) if st.num_questions else 8))
    pq = W.prefill_queries(st)
    iq = None if ins is None else W.instruction_queries(st, ins)
    q_ctx, q_seg = db.pack_prefill_queries(pq.ctx_q, pq.seg_q, st.seg_len0, instr_q=iq)
    oc, os_ = db.prefill_outputs(fill=SENTINEL)
    bound = max([int(st.seg_len0[st.q_start[b]:st.q_start[b + 1]].sum()) for b in range(wl.num_prompts)] + [0])
    standard = cfg["mode"] == "standard"
    db.prefill(0, q_ctx, q_seg, oc, os_, bound, standard=standard)
    torch.cuda.synchronize()
    oc_h, os_h = oc.cpu().numpy(), os_.cpu().numpy()
    refs = P.prefill_standard(kv.ctx_k, kv.ctx_v, pq.ctx_q, st.ctx_start, st.q_start, kv.seg_k, kv.seg_v, pq.seg_q,
                              st.seg_start, wl.rope_base,
                              instr=None if ins is None else (ins.prompt_start, ins.tok_start, ins.k, ins.v, iq))
    r_ctx, r_seg = refs[0], refs[1]
    errs = []
    for b in range(wl.num_prompts):
        if standard and st.q_count[b] == 0:
            continue                                  # no question's prompt holds this context
        rows = oc_h[db.ctx_off[b]: db.ctx_off[b] + st.ctx_len[b]]
        errs.append(max_err(rows, r_ctx[st.ctx_start[b]: st.ctx_start[b + 1]]) if len(rows) else 0.0)
    for i in range(st.num_questions):
        s = int(st.seg_len0[i])
        if s:
            errs.append(max_err(os_h[i, :s], r_seg[st.seg_start[i]: st.seg_start[i + 1]]))
    if ins is not None:
        r_ins = refs[2]
        for s_ in range(len(ins.lp)):
            nq = int(st.q_start[ins.prompt_start[s_ + 1]] - st.q_start[ins.prompt_start[s_]])
            if standard and nq == 0:
                continue
            n = int(ins.lp[s_])
            if n:
                errs.append(max_err(oc_h[db.instr_off[s_]: db.instr_off[s_] + n],
                                    r_ins[ins.tok_start[s_]: ins.tok_start[s_ + 1]]))
    e = max(errs + [0.0])
    log(f"  max err {e:.3e} over {len(errs)} row blocks")
    assert e <= tol(wl.dtype)
    assert db.err_flag() == 0
