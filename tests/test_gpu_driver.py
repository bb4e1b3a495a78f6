"""GPU: the multi-step, multi-layer decode loop, eager and replayed from a HIP
graph.  A graph replay runs the kernels of the eager sequence with the same
arguments, so its outputs must equal the eager run's bit for bit; the eager
run itself is checked against the fp64 oracle at its last step.  Covered:
the fused step (IPPD and the standard baseline), a two-level batch, the
dense-mask baseline, and a prefill call."""
import numpy as np
import pytest
import torch

import workload as W
from oracle import ippd as O
from oracle import prefill as P
from paper_2609_05707_amd.driver import DecodeLoop
from paper_2609_05707_amd.session import DecodeBatch
from tests.gpu_harness import load_layer, log, make_batch, max_err, oracle_steps

pytestmark = pytest.mark.gpu


def _loop(st, layers, standard=False, dense=False, ins=None):
    if ins is None:
        db = make_batch(st, layers=layers)
    else:
        wl = st.wl
        db = DecodeBatch(st.ctx_len.tolist(), st.q_count.tolist(), wl.hq, wl.hkv, wl.head_dim, wl.dtype,
                         int(st.seg_len0.max()) + wl.steps, rope_base=wl.rope_base, layers=layers,
                         instr_len=ins.lp.tolist(), instr_prompt_start=ins.prompt_start.tolist())
    kv = W.layer_kv(st)
    for l in range(layers):
        if ins is not None:
            db.load_instructions(l, ins.k, ins.v)
        load_layer(db, st, l, kv)
    q, k, v, act = [], [], [], []
    for t in range(st.wl.steps):
        si = W.step_inputs(st, t)
        q.append(db.to_dev(si.q_new)); k.append(db.to_dev(si.k_new)); v.append(db.to_dev(si.v_new))
        act.append(torch.from_numpy(si.active.astype(np.uint8)).to(db.device))
    return DecodeLoop(db, q, k, v, act, standard=standard, dense=dense), kv


def _replays_equal_eager(loop, layers, eager_out, eager_seg, reps=3):
    """Three replays, each bit-equal to the eager run, with eager work on the
    same stream and buffers between them."""
    db = loop.db
    loop.capture()
    for rep in range(reps):
        loop.reset()
        db.out.fill_(-5.0)
        loop.replay()
        torch.cuda.synchronize()
        assert torch.equal(db.out, eager_out), f"replay {rep} differs from the eager run"
        for l in range(layers):
            assert torch.equal(db.seg_len[l], eager_seg[l])
        loop.reset()
        loop.enqueue(steps=1)
        torch.cuda.synchronize()


@pytest.mark.parametrize("standard", [False, True])
def test_graph_replay_equals_eager_and_oracle(standard):
    log(f"case: decode loop, 4 steps x 3 layers, graph replay vs eager (standard={standard})")
    wl = W.custom_workload(wid=250, dtype="bf16", num_prompts=3, hq=8, hkv=2, head_dim=128,
                           ctx_len=(100, 400), questions=(2, 7), seg_len=(3, 40), steps=4,
                           stop=(2, 4), value_std=0.5)
    st = W.make_structure(wl)
    loop, kv = _loop(st, layers=3, standard=standard)
    db = loop.db
    loop.reset()
    db.out.fill_(-5.0)
    loop.enqueue()
    torch.cuda.synchronize()
    eager_out = db.out.clone()
    eager_seg = [db.seg_len[l].clone() for l in range(3)]
    # the last step's rows of active questions against the oracle
    last = wl.steps - 1
    ref = oracle_steps(st, kv, list(range(wl.steps)), [last])[last]
    act = st.active(last)
    got = eager_out[: st.num_questions].float().cpu().numpy()
    e = max_err(got[act], ref[0][act])
    log(f"eager last step max err {e:.3e}")
    assert e <= 2e-2
    np.testing.assert_array_equal(eager_seg[0][: st.num_questions].cpu().numpy(), st.seg_len_at(wl.steps))

    loop.capture()
    for rep in range(3):
        loop.reset()
        db.out.fill_(-5.0)
        loop.replay()
        torch.cuda.synchronize()
        assert torch.equal(db.out, eager_out), f"replay {rep} differs from the eager run"
        for l in range(3):
            assert torch.equal(db.seg_len[l], eager_seg[l])
        # eager work between replays on the same stream and buffers
        loop.reset()
        loop.enqueue(steps=1)
        torch.cuda.synchronize()
    assert db.err_flag() == 0


def _eager(loop, layers):
    db = loop.db
    loop.reset()
    db.out.fill_(-5.0)
    loop.enqueue()
    torch.cuda.synchronize()
    return db.out.clone(), [db.seg_len[l].clone() for l in range(layers)]


@pytest.mark.parametrize("standard", [False, True])
def test_graph_replay_two_level(standard):
    """A two-level batch (instruction units and instruction merge slots) in the
    loop: eager against the oracle at the last step, replays bit-equal."""
    log(f"case: two-level decode loop, 3 steps x 2 layers, graph replay (standard={standard})")
    wl = W.custom_workload(wid=251, dtype="bf16", num_prompts=4, hq=8, hkv=2, head_dim=128,
                           ctx_len=(60, 300), questions=(1, 5), seg_len=(2, 30), steps=3,
                           stop=(2, 3), value_std=0.5)
    st = W.make_structure(wl)
    ins = W.instructions(st, 2, (200, 700))
    loop, kv = _loop(st, layers=2, standard=standard, ins=ins)
    eager_out, eager_seg = _eager(loop, 2)
    state = O.KVState.from_packed(kv.seg_k, kv.seg_v, st.seg_start)
    instr = O.Instructions(ins.prompt_start, ins.tok_start, ins.k, ins.v)
    for t in range(wl.steps):
        si = W.step_inputs(st, t)
        if t == wl.steps - 1:
            ref, _ = O.decode_step_standard(kv.ctx_k, kv.ctx_v, st.ctx_start, st.q_start, state, si.q_new,
                                            si.k_new, si.v_new, si.active, wl.rope_base, instr=instr)
        state.append(si.k_new, si.v_new, si.active)
    act = st.active(wl.steps - 1)
    e = max_err(eager_out[: st.num_questions].float().cpu().numpy()[act], ref[act])
    log(f"eager last step max err {e:.3e}")
    assert e <= 2e-2
    _replays_equal_eager(loop, 2, eager_out, eager_seg)
    assert loop.db.err_flag() == 0


def test_graph_replay_dense_baseline():
    """The dense-mask baseline as append + dense decode calls in the loop."""
    log("case: dense-mask baseline loop, 3 steps x 2 layers, graph replay")
    wl = W.custom_workload(wid=252, dtype="bf16", num_prompts=3, hq=8, hkv=2, head_dim=128,
                           ctx_len=(100, 400), questions=(2, 7), seg_len=(3, 40), steps=3,
                           stop=(2, 3), value_std=0.5)
    st = W.make_structure(wl)
    loop, kv = _loop(st, layers=2, dense=True)
    eager_out, eager_seg = _eager(loop, 2)
    last = wl.steps - 1
    ref = oracle_steps(st, kv, list(range(wl.steps)), [last])[last]
    act = st.active(last)
    e = max_err(eager_out[: st.num_questions].float().cpu().numpy()[act], ref[0][act])
    log(f"eager last step max err {e:.3e}")
    assert e <= 2e-2
    _replays_equal_eager(loop, 2, eager_out, eager_seg)
    assert loop.db.err_flag() == 0


def test_graph_replay_prefill():
    """A prefill call (IPPD, then the baseline) captured once and replayed:
    every replay bit-equal to the eager call, the eager call against the oracle."""
    log("case: prefill graph replay")
    wl = W.custom_workload(wid=253, dtype="bf16", num_prompts=3, hq=8, hkv=2, head_dim=128, ctx_len=(50, 300),
                           questions=(1, 4), question_tokens=0, seg_len=(1, 40), value_std=0.5)
    st = W.make_structure(wl)
    kv = W.layer_kv(st)
    pq = W.prefill_queries(st)
    db = DecodeBatch(st.ctx_len.tolist(), st.q_count.tolist(), wl.hq, wl.hkv, wl.head_dim, wl.dtype,
                     max(8, int(st.seg_len0.max())), rope_base=wl.rope_base)
    load_layer(db, st, 0, kv)
    q_ctx, q_seg = db.pack_prefill_queries(pq.ctx_q, pq.seg_q, st.seg_len0)
    oc, os_ = db.prefill_outputs(fill=-5.0)
    bound = max(int(st.seg_len0[st.q_start[b]:st.q_start[b + 1]].sum()) for b in range(wl.num_prompts))
    r_ctx, r_seg = P.prefill_standard(kv.ctx_k, kv.ctx_v, pq.ctx_q, st.ctx_start, st.q_start, kv.seg_k, kv.seg_v,
                                      pq.seg_q, st.seg_start, wl.rope_base)
    for standard in (False, True):
        oc.fill_(-5.0)
        os_.fill_(-5.0)
        db.prefill(0, q_ctx, q_seg, oc, os_, bound, standard=standard)
        torch.cuda.synchronize()
        e_oc, e_os = oc.clone(), os_.clone()
        g_ctx = np.concatenate([e_oc.cpu().numpy()[db.ctx_off[b]: db.ctx_off[b] + st.ctx_len[b]]
                                for b in range(wl.num_prompts)])
        e = max_err(g_ctx, r_ctx)
        log(f"eager prefill (standard={standard}) context rows max err {e:.3e}")
        assert e <= 2e-2
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g):
            db.prefill(0, q_ctx, q_seg, oc, os_, bound, standard=standard)
        torch.cuda.synchronize()
        for rep in range(3):
            oc.fill_(-5.0)
            os_.fill_(-5.0)
            g.replay()
            torch.cuda.synchronize()
            assert torch.equal(oc, e_oc) and torch.equal(os_, e_os), f"replay {rep} differs"
            db.prefill(0, q_ctx, q_seg, oc, os_, bound, standard=not standard)   # eager work between replays
            torch.cuda.synchronize()
    assert db.err_flag() == 0
