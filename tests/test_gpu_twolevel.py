"""GPU: two-level batches (Sec. 4.4: several contexts behind one instruction p,
which is read once for all their questions) against the fp64 oracle over
several decode steps, for the fused step (append + attention), the separate
calls and the standard baseline; and equality with the one-level layout in
which every context carries its own copy of the instruction.  Tolerances:
1e-5 for fp32, 2e-2 for bf16."""
import numpy as np
import pytest
import torch

import workload as W
from oracle import ippd as O
from paper_2609_05707_amd.session import DecodeBatch
from tests.gpu_harness import log, max_err

pytestmark = pytest.mark.gpu

SENTINEL = -555.0


def tol(dtype):
    return 1e-5 if dtype == "f32" else 2e-2


def build(st, ins, chunk_tokens=0, extra=8):
    wl = st.wl
    cap = int(st.seg_len0.max()) + wl.steps + extra
    db = DecodeBatch(st.ctx_len.tolist(), st.q_count.tolist(), wl.hq, wl.hkv, wl.head_dim, wl.dtype, cap,
                     rope_base=wl.rope_base, chunk_tokens=chunk_tokens, instr_len=ins.lp.tolist(),
                     instr_prompt_start=ins.prompt_start.tolist())
    kv = W.layer_kv(st)
    db.load_instructions(0, ins.k, ins.v)
    db.load_context(0, kv.ctx_k, kv.ctx_v)
    db.load_segments(0, kv.seg_k, kv.seg_v, st.seg_len0)
    return db, kv


def run_steps(db, st, mode):
    outs = []
    for t in range(st.wl.steps):
        si = W.step_inputs(st, t)
        db.set_active(si.active)
        q, k, v = db.to_dev(si.q_new), db.to_dev(si.k_new), db.to_dev(si.v_new)
        db.out.fill_(SENTINEL)
        if mode == "fused":
            db.decode_step(0, q, k, v)
        elif mode == "separate":
            db.append(0, q, k, v)
            db.decode(0)
        else:
            db.decode_step(0, q, k, v, standard=True)
        torch.cuda.synchronize()
        outs.append(db.out[: st.num_questions].cpu().numpy().copy())
    return outs


CASES = [
    # name, dtype, hq, hkv, D, B, ctx, questions, seg, stop, contexts per instruction, instruction length, chunk
    ("bf16-cpi2", "bf16", 8, 2, 128, 5, (30, 200), (0, 4), (3, 40), (1, 3), 2, (0, 300), 0),
    ("bf16-long-instr", "bf16", 8, 2, 128, 6, (200, 600), (2, 6), (8, 40), None, 3, (1500, 2500), 256),
    ("f32-one-instr", "f32", 4, 2, 64, 4, (40, 120), (1, 3), (2, 20), None, 4, (100, 200), 0),
]


@pytest.mark.parametrize("mode", ["fused", "separate", "standard"])
@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_two_level_decode_parity(case, mode):
    name, dtype, hq, hkv, d, B, ctx, qs, seg, stop, cpi, lp, chunk = case
    log(f"case: two-level {name} mode={mode}")
    wl = W.custom_workload(wid=600 + CASES.index(case), dtype=dtype, num_prompts=B, hq=hq, hkv=hkv, head_dim=d,
                           ctx_len=ctx, questions=qs, seg_len=seg, steps=3, stop=stop,
                           value_std=0.5 if dtype == "bf16" else 1.0)
    st = W.make_structure(wl)
    ins = W.instructions(st, cpi, lp)
    db, kv = build(st, ins, chunk_tokens=chunk)
    got = run_steps(db, st, mode)
    instr = O.Instructions(ins.prompt_start, ins.tok_start, ins.k, ins.v)
    state = O.KVState.from_packed(kv.seg_k, kv.seg_v, st.seg_start)
    for t in range(wl.steps):
        si = W.step_inputs(st, t)
        ref, _ = O.decode_step_standard(kv.ctx_k, kv.ctx_v, st.ctx_start, st.q_start, state, si.q_new, si.k_new,
                                        si.v_new, si.active, wl.rope_base, instr=instr)
        state.append(si.k_new, si.v_new, si.active)
        act = si.active
        e = max_err(got[t][act], ref[act])
        log(f"  step {t}: {int(act.sum())} active, max err {e:.3e}")
        assert e <= tol(dtype)
        assert (got[t][~act] == SENTINEL).all()
    np.testing.assert_array_equal(db.seg_len[0][: st.num_questions].cpu().numpy(), st.seg_len_at(wl.steps))
    assert db.err_flag() == 0


def test_two_level_equals_folded_instruction():
    """Reading p once for all contexts gives the result of the one-level
    layout in which each context is p followed by c_b (the same keys at the
    same positions), to within the bf16 rounding of the two paths."""
    log("case: two-level vs folded one-level")
    wl = W.custom_workload(wid=620, dtype="bf16", num_prompts=4, hq=8, hkv=2, head_dim=128, ctx_len=(50, 150),
                           questions=(1, 4), seg_len=(4, 30), steps=2, value_std=0.5)
    st = W.make_structure(wl)
    ins = W.instructions(st, 2, (100, 400))
    db2, kv = build(st, ins)
    two = run_steps(db2, st, "fused")
    # one-level: context b := [instruction of b; c_b]
    s_of = np.searchsorted(ins.prompt_start, np.arange(wl.num_prompts), side="right") - 1
    fk, fv, flen = [], [], []
    for b in range(wl.num_prompts):
        i0, i1 = ins.tok_start[s_of[b]], ins.tok_start[s_of[b] + 1]
        c0, c1 = st.ctx_start[b], st.ctx_start[b + 1]
        fk.append(np.concatenate([ins.k[i0:i1], kv.ctx_k[c0:c1]]))
        fv.append(np.concatenate([ins.v[i0:i1], kv.ctx_v[c0:c1]]))
        flen.append(len(fk[-1]))
    db1 = DecodeBatch(flen, st.q_count.tolist(), wl.hq, wl.hkv, wl.head_dim, wl.dtype,
                      int(st.seg_len0.max()) + wl.steps + 8, rope_base=wl.rope_base)
    db1.load_context(0, np.concatenate(fk), np.concatenate(fv))
    db1.load_segments(0, kv.seg_k, kv.seg_v, st.seg_len0)
    one = run_steps(db1, st, "fused")
    for t in range(wl.steps):
        act = W.step_inputs(st, t).active
        e = float(np.max(np.abs(two[t][act] - one[t][act])))
        log(f"  step {t}: max |two-level - folded| = {e:.3e}")
        assert e <= 2e-2
    assert db1.err_flag() == 0 and db2.err_flag() == 0


@pytest.mark.parametrize("fault", ["misaligned-offset", "length-over-bound"])
def test_bad_instruction_layout_is_flagged(fault):
    """A two-level batch whose instruction table breaks the layout (an offset not
    a multiple of 8, or a length above max_instr_len) is caught by the kernels'
    own checks before any access with it: the decode step and both prefill
    modes raise IPPD_FLAG_BAD_LAYOUT and every kernel exits normally."""
    from paper_2609_05707_amd import _lib as L
    log(f"case: two-level bad instruction layout ({fault})")
    wl = W.custom_workload(wid=630, dtype="bf16", num_prompts=3, hq=8, hkv=2, head_dim=128, ctx_len=(40, 120),
                           questions=(1, 3), seg_len=(2, 20), steps=1, value_std=0.5)
    st = W.make_structure(wl)
    ins = W.instructions(st, 2, (50, 150))
    db, kv = build(st, ins)
    if fault == "misaligned-offset":
        db.d_instr_off[1] = int(db.instr_off[1]) + 3
    else:
        db.d_instr_len[0] = int(ins.lp.max()) + 8
    torch.cuda.synchronize()
    si = W.step_inputs(st, 0)
    db.set_active(si.active)
    seg0 = db.seg_len[0].clone()
    for standard in (False, True):
        # a broken instruction table leaves every question unserved: no row is
        # formed from instruction slots the instruction units did not write
        db.seg_len[0].copy_(seg0)
        db.d_err.zero_()
        db.out.fill_(SENTINEL)
        db.ws_ippd.fill_(0xFF)
        db.ws_std.fill_(0xFF)
        db.decode_step(0, db.to_dev(si.q_new), db.to_dev(si.k_new), db.to_dev(si.v_new), standard=standard)
        torch.cuda.synchronize()
        assert db.err_flag() & L.IPPD_FLAG_BAD_LAYOUT, standard
        assert np.all(db.out[: st.num_questions].cpu().numpy() == SENTINEL), standard
    pq = W.prefill_queries(st)
    iq = W.instruction_queries(st, ins)
    q_ctx, q_seg = db.pack_prefill_queries(pq.ctx_q, pq.seg_q, st.seg_len0, instr_q=iq)
    oc, os_ = db.prefill_outputs()
    for standard in (False, True):
        db.d_err.zero_()
        db.prefill(0, q_ctx, q_seg, oc, os_, int(st.seg_len0.sum()), standard=standard)
        torch.cuda.synchronize()
        assert db.err_flag() & L.IPPD_FLAG_BAD_LAYOUT, standard
