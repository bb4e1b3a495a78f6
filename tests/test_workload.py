"""The seeded input generator: determinism, ranges, bf16 rounding."""
import numpy as np
import pytest
import torch

import workload as W


def test_bf16_rounding_matches_torch():
    x = np.random.default_rng(0).standard_normal(100000).astype(np.float32) * 3
    x[:4] = [1.0 + 2**-8, 1.0 + 3 * 2**-8, -1.0 - 2**-8, 0.0]     # ties
    ours = W.round_to_bf16(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float32).numpy()
    np.testing.assert_array_equal(ours, ref)
    bits = W.bf16_bits(ours)
    back = torch.from_numpy(bits.view(np.int16)).view(torch.bfloat16).float().numpy()
    np.testing.assert_array_equal(back, ours)


@pytest.mark.parametrize("wid", [1, 2, 3, 4, 5])
def test_structure_ranges(wid):
    wl = W.workload(wid)
    st = W.make_structure(wl)
    assert len(st.ctx_len) == wl.num_prompts
    assert ((st.ctx_len >= wl.ctx_len[0]) & (st.ctx_len <= wl.ctx_len[1])).all()
    assert ((st.q_count >= wl.questions[0]) & (st.q_count <= wl.questions[1])).all()
    lo = wl.question_tokens + wl.seg_len[0]
    hi = wl.question_tokens + wl.seg_len[1]
    assert ((st.seg_len0 >= lo) & (st.seg_len0 <= hi)).all()
    assert st.num_questions == st.q_count.sum()
    if wl.stop is None:
        assert st.active(wl.steps - 1).all()
    else:
        assert ((st.stop >= wl.stop[0]) & (st.stop <= wl.stop[1])).all()


def test_fixed_shapes_of_named_workloads():
    st = W.make_structure(W.workload(1))
    assert list(st.ctx_len) == [256] and list(st.seg_len0) == [24] * 4
    st2 = W.make_structure(W.workload(2))
    assert st2.num_questions == 16 and st2.ctx_len[0] == 4096
    st5 = W.make_structure(W.workload(5))
    assert (st5.seg_len0 == 32).all() and st5.num_questions == 256


def test_determinism_and_layer_independence():
    wl = W.workload(1)
    st = W.make_structure(wl)
    a, b = W.layer_kv(st, 0), W.layer_kv(st, 0)
    np.testing.assert_array_equal(a.ctx_k, b.ctx_k)
    c = W.layer_kv(st, 1)
    assert not np.array_equal(a.ctx_k, c.ctx_k)
    s0, s0b = W.step_inputs(st, 0), W.step_inputs(st, 0)
    np.testing.assert_array_equal(s0.q_new, s0b.q_new)
    assert a.ctx_k.dtype == np.float32 and a.ctx_k.shape == (256, 2, 64)


def test_bf16_workload_values_are_bf16():
    wl = W.custom_workload(dtype="bf16", value_std=0.5)
    st = W.make_structure(wl)
    kv = W.layer_kv(st)
    np.testing.assert_array_equal(W.round_to_bf16(kv.ctx_k), kv.ctx_k)
