"""GPU: the multi-step, multi-layer decode loop, eager and replayed from a HIP
graph.  A graph replay runs the kernels of the eager sequence with the same
arguments, so its outputs must equal the eager run's bit for bit; the eager
run itself is checked against the fp64 oracle at its last step."""
import numpy as np
import pytest
import torch

import workload as W
from paper_2609_05707_amd.driver import DecodeLoop
from tests.gpu_harness import load_layer, log, make_batch, max_err, oracle_steps

pytestmark = pytest.mark.gpu


def _loop(st, layers, standard=False):
    db = make_batch(st, layers=layers)
    kv = W.layer_kv(st)
    for l in range(layers):
        load_layer(db, st, l, kv)
    q, k, v, act = [], [], [], []
    for t in range(st.wl.steps):
        si = W.step_inputs(st, t)
        q.append(db.to_dev(si.q_new)); k.append(db.to_dev(si.k_new)); v.append(db.to_dev(si.v_new))
        act.append(torch.from_numpy(si.active.astype(np.uint8)).to(db.device))
    return DecodeLoop(db, q, k, v, act, standard=standard), kv


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
