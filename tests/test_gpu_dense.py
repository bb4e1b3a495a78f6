"""GPU: the dense-mask baseline (dense_decode_attention: the paper's own
scheme, every new-token row over all keys of its stacked prompt under M_fin)
against the fp64 oracle over several decode steps with a shrinking active
set, and against the block-diagonal IPPD attention on the same inputs.
Tolerances: 1e-5 for fp32, 2e-2 for bf16."""
import numpy as np
import pytest
import torch

import workload as W
from oracle import ippd as O
from tests.gpu_harness import load_layer, log, make_batch, max_err

pytestmark = pytest.mark.gpu

SENTINEL = -333.0

CASES = [
    # name, dtype, hq, hkv, D, B, ctx, questions, seg, stop, chunk
    ("bf16-d128-g4", "bf16", 8, 2, 128, 3, (40, 400), (1, 6), (3, 70), (1, 3), 0),
    ("bf16-d128-g4-rows128", "bf16", 8, 2, 128, 2, (100, 300), (20, 32), (1, 40), (2, 3), 128),
    ("bf16-d64-g2", "bf16", 4, 2, 64, 2, (30, 200), (1, 5), (2, 50), None, 0),
    ("f32-d128-g4", "f32", 8, 2, 128, 2, (33, 150), (1, 4), (1, 33), (1, 3), 0),
    ("f32-d64-g1", "f32", 2, 2, 64, 3, (1, 90), (0, 4), (1, 45), None, 64),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_dense_mask_parity(case):
    name, dtype, hq, hkv, d, B, ctx, qs, seg, stop, chunk = case
    log(f"case: dense-mask {name}")
    wl = W.custom_workload(wid=800 + CASES.index(case), dtype=dtype, num_prompts=B, hq=hq, hkv=hkv, head_dim=d,
                           ctx_len=ctx, questions=qs, seg_len=seg, steps=3, stop=stop,
                           value_std=0.5 if dtype == "bf16" else 1.0)
    st = W.make_structure(wl)
    kv = W.layer_kv(st)
    db = make_batch(st, chunk_tokens=chunk)
    load_layer(db, st, 0, kv)
    state = O.KVState.from_packed(kv.seg_k, kv.seg_v, st.seg_start)
    tol = 1e-5 if dtype == "f32" else 2e-2
    out_ippd = torch.empty_like(db.out)
    for t in range(wl.steps):
        si = W.step_inputs(st, t)
        db.set_active(si.active)
        db.append(0, db.to_dev(si.q_new), db.to_dev(si.k_new), db.to_dev(si.v_new))
        db.out.fill_(SENTINEL)
        db.decode(0, dense=True)
        db.decode(0, out=out_ippd, lse=torch.empty_like(db.lse))
        torch.cuda.synchronize()
        got = db.out[: st.num_questions].cpu().numpy()
        ref, _ = O.decode_step_standard(kv.ctx_k, kv.ctx_v, st.ctx_start, st.q_start, state, si.q_new, si.k_new,
                                        si.v_new, si.active, wl.rope_base)
        state.append(si.k_new, si.v_new, si.active)
        act = si.active
        e = max_err(got[act], ref[act])
        e_ippd = float(np.max(np.abs(got[act] - out_ippd[: st.num_questions].cpu().numpy()[act]))) if act.any() else 0.0
        log(f"  step {t}: {int(act.sum())} active, max err {e:.3e}, max |dense - ippd| {e_ippd:.3e}")
        assert e <= tol and e_ippd <= tol
        assert (got[~act] == SENTINEL).all()
    assert db.err_flag() == 0
