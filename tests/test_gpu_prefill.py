"""GPU: stacked-prompt prefill attention (ippd_prefill_attention and the
standard baseline) against the fp64 oracle, element by element, on seeded
ragged inputs that span several tiles and ragged tails, with sentinels on
every row the library must not write; plus sampled rows at a
Llama-3-8B-shaped size.  Tolerances: 1e-5 for fp32, 2e-2 for bf16 (inputs
rounded to bf16 on both sides; the kernels round rotated queries and the
softmax weights to bf16 for the MFMA products, accumulate in fp32)."""
import numpy as np
import pytest
import torch

import workload as W
from oracle import prefill as P
from paper_2609_05707_amd import _lib as L
from paper_2609_05707_amd.session import DecodeBatch
from tests.gpu_harness import log, max_err

pytestmark = pytest.mark.gpu

SENTINEL = -777.0


def tol(dtype):
    return 1e-5 if dtype == "f32" else 2e-2


def prefill_case(wl, standard=False, bound=None, ctx_rows=None, seg_rows=None, tile_rows=0):
    """Run one prefill on the GPU; return (structure, gpu_ctx, gpu_seg, ref_ctx, ref_seg, db, oc, os)
    with GPU rows gathered into the oracle's packed order.  tile_rows 128 / 256 fixes
    the unit size of the bf16 D = 128 kernel (0: the planner's choice)."""
    st = W.make_structure(wl)
    kv = W.layer_kv(st)
    pq = W.prefill_queries(st)
    cap = max(8, int(st.seg_len0.max()) if st.num_questions else 8)
    db = DecodeBatch(st.ctx_len.tolist(), st.q_count.tolist(), wl.hq, wl.hkv, wl.head_dim, wl.dtype, cap,
                     rope_base=wl.rope_base, tile_rows=tile_rows)
    db.load_context(0, kv.ctx_k, kv.ctx_v)
    db.load_segments(0, kv.seg_k, kv.seg_v, st.seg_len0)
    q_ctx, q_seg = db.pack_prefill_queries(pq.ctx_q, pq.seg_q, st.seg_len0)
    oc, os_ = db.prefill_outputs(fill=SENTINEL)
    if bound is None:
        per_prompt = [int(st.seg_len0[st.q_start[b]:st.q_start[b + 1]].sum()) for b in range(wl.num_prompts)]
        bound = max(per_prompt + [0])
    db.prefill(0, q_ctx, q_seg, oc, os_, bound, standard=standard)
    torch.cuda.synchronize()
    oc_h, os_h = oc.cpu().numpy(), os_.cpu().numpy()
    g_ctx = np.concatenate([oc_h[db.ctx_off[b]: db.ctx_off[b] + st.ctx_len[b]] for b in range(wl.num_prompts)])
    g_seg = (np.concatenate([os_h[i, : st.seg_len0[i]] for i in range(st.num_questions)])
             if st.num_questions else np.zeros((0, wl.hq, wl.head_dim)))
    r_ctx, r_seg = P.prefill_standard(kv.ctx_k, kv.ctx_v, pq.ctx_q, st.ctx_start, st.q_start, kv.seg_k, kv.seg_v,
                                      pq.seg_q, st.seg_start, wl.rope_base, ctx_rows=ctx_rows, seg_rows=seg_rows)
    return st, g_ctx, g_seg, r_ctx, r_seg, db, oc_h, os_h


def check_unwritten(st, db, oc_h, os_h, standard=False):
    """Pool rows outside every context and segment slots past the question stay untouched."""
    written = np.zeros(db.pool, bool)
    for b in range(len(st.ctx_len)):
        if standard and st.q_count[b] == 0:
            continue
        written[db.ctx_off[b]: db.ctx_off[b] + st.ctx_len[b]] = True
    assert (oc_h[~written] == SENTINEL).all()
    for i in range(st.num_questions):
        assert (os_h[i, st.seg_len0[i]:] == SENTINEL).all()


CASES = [
    # (name, dtype, hq, hkv, D, B, ctx range, questions range, question-token range)
    ("bf16-d128-g4", "bf16", 8, 2, 128, 3, (40, 300), (0, 5), (1, 40)),
    ("bf16-d128-g1", "bf16", 4, 4, 128, 2, (1, 90), (1, 3), (0, 70)),
    ("bf16-d128-g3", "bf16", 12, 4, 128, 2, (100, 200), (2, 4), (3, 50)),
    ("bf16-d128-g16", "bf16", 32, 2, 128, 2, (30, 150), (1, 3), (1, 20)),
    ("bf16-d64-g4", "bf16", 8, 2, 64, 2, (50, 260), (1, 4), (1, 36)),
    ("f32-d128-g4", "f32", 8, 2, 128, 2, (33, 170), (1, 4), (1, 33)),
    ("f32-d64-g2", "f32", 4, 2, 64, 3, (1, 200), (0, 3), (0, 45)),
]


def _with_unit_sizes(cases, dtype_at, d_at, sizes):
    """(case, tile_rows) pairs: the bf16 D = 128 kernel at each unit size, the
    others (one unit size) once."""
    out = []
    for c in cases:
        for r in (sizes if (c[dtype_at] == "bf16" and c[d_at] == 128) else [0]):
            out.append(pytest.param(c, r, id=f"{c[0]}-rows{r}"))
    return out


@pytest.mark.parametrize("standard", [False, True])
@pytest.mark.parametrize("case,rows", _with_unit_sizes(CASES, 1, 4, [0, 128, 256]))
def test_prefill_parity(case, rows, standard):
    name, dtype, hq, hkv, d, B, ctx, qs, ql = case
    log(f"case: prefill {name} standard={standard} tile_rows={rows}")
    wl = W.custom_workload(wid=400 + CASES.index(case), dtype=dtype, num_prompts=B, hq=hq, hkv=hkv, head_dim=d,
                           ctx_len=ctx, questions=qs, question_tokens=0, seg_len=ql, value_std=0.5 if dtype == "bf16" else 1.0)
    st, g_ctx, g_seg, r_ctx, r_seg, db, oc_h, os_h = prefill_case(wl, standard=standard, tile_rows=rows)
    if standard:
        # standard prompting runs one prompt per question: the context of a prompt
        # without questions is never prefilled, and its rows stay untouched
        for b in np.flatnonzero(st.q_count == 0):
            rows = slice(st.ctx_start[b], st.ctx_start[b + 1])
            assert (g_ctx[rows] == SENTINEL).all()
            r_ctx[rows] = np.nan
    e_ctx, e_seg = max_err(g_ctx, r_ctx), max_err(g_seg, r_seg)
    log(f"  ctx rows {len(g_ctx)} max err {e_ctx:.3e}; question rows {len(g_seg)} max err {e_seg:.3e}")
    assert e_ctx <= tol(dtype) and e_seg <= tol(dtype)
    check_unwritten(st, db, oc_h, os_h, standard)
    assert db.err_flag() == 0


def test_ippd_and_standard_agree_closely():
    """The two paths run the same per-row arithmetic over the same visible keys
    (masked tiles add exact zeros), so they agree far inside the tolerance."""
    log("case: prefill ippd vs standard")
    wl = W.custom_workload(wid=420, dtype="bf16", num_prompts=2, hq=8, hkv=2, head_dim=128, ctx_len=(60, 200),
                           questions=(2, 5), question_tokens=0, seg_len=(1, 40))
    a = prefill_case(wl, standard=False)
    b = prefill_case(wl, standard=True)
    assert np.max(np.abs(a[1] - b[1])) <= 1e-6
    assert np.max(np.abs(a[2] - b[2])) <= 1e-6


def test_prefill_full_size_sampled():
    """Llama-3-8B-shaped prompt (Hq 32, Hkv 8, D 128, bf16), context 4096, 16
    questions of 32 tokens: sampled rows against the oracle, computed row by row."""
    log("case: prefill llama3-8b lc4096 n16 q32, sampled rows")
    wl = W.custom_workload(wid=430, name="prefill-llama3-8b-lc4096-n16", dtype="bf16", num_prompts=1, hq=32,
                           hkv=8, head_dim=128, ctx_len=(4096, 4096), questions=(16, 16), question_tokens=32,
                           seg_len=(0, 0), value_std=0.5)
    rng = np.random.default_rng(7)
    ctx_rows = sorted(set([0, 1, 31, 32, 63, 64, 4095] + rng.integers(0, 4096, 20).tolist()))
    seg_rows = sorted(set([0, 31, 32, 511] + rng.integers(0, 512, 12).tolist()))
    st, g_ctx, g_seg, r_ctx, r_seg, db, oc_h, os_h = prefill_case(wl, ctx_rows=ctx_rows, seg_rows=seg_rows)
    e_ctx = max_err(g_ctx[ctx_rows], r_ctx[ctx_rows])
    e_seg = max_err(g_seg[seg_rows], r_seg[seg_rows])
    log(f"  sampled ctx max err {e_ctx:.3e}, question max err {e_seg:.3e}")
    assert e_ctx <= 2e-2 and e_seg <= 2e-2
    assert np.isfinite(g_ctx).all() and np.isfinite(g_seg).all()
    assert db.err_flag() == 0


def test_question_bound_violation_is_flagged():
    """A prompt with more question tokens than the caller's bound sets
    IPPD_FLAG_BAD_LAYOUT (the kernel only skips rows; every wave exits normally)."""
    log("case: prefill bound violation")
    wl = W.custom_workload(wid=440, dtype="bf16", num_prompts=1, hq=8, hkv=2, head_dim=128, ctx_len=(64, 64),
                           questions=(4, 4), question_tokens=40, seg_len=(0, 0))
    st, g_ctx, g_seg, r_ctx, r_seg, db, oc_h, os_h = prefill_case(wl, bound=20)
    assert db.err_flag() & L.IPPD_FLAG_BAD_LAYOUT
    assert max_err(g_ctx, r_ctx) <= 2e-2                       # context rows are unaffected


TWO_LEVEL = [
    # (name, seed, dtype, hq, hkv, D, B, ctx range, questions range, question tokens,
    #  contexts per instruction, |p| range)
    ("bf16-d128-cpi2", 450, "bf16", 8, 2, 128, 5, (30, 200), (0, 4), (1, 40), 2, (0, 300)),
    ("bf16-d64-long-instr", 451, "bf16", 8, 2, 64, 4, (1, 90), (1, 3), (0, 30), 3, (100, 400)),
    ("f32-d128-cpi2", 452, "f32", 8, 2, 128, 3, (20, 100), (1, 3), (1, 20), 2, (40, 150)),
    ("f32-d64-one-instr", 453, "f32", 4, 2, 64, 3, (10, 70), (0, 3), (1, 25), 3, (1, 90)),
    # |p| = 52, 60, 6, 0 with 1, 0, 2, 2 questions: an instruction nobody asks
    # about (the baseline leaves its rows) and an empty instruction
    ("f32-d64-cpi1-empty", 463, "f32", 4, 2, 64, 4, (10, 70), (0, 2), (1, 25), 1, (0, 60)),
]


@pytest.mark.parametrize("standard", [False, True])
@pytest.mark.parametrize("case,rows", _with_unit_sizes(TWO_LEVEL, 2, 5, [0, 256]))
def test_two_level_prefill_parity(case, rows, standard):
    """Two-level batch (Sec. 4.4): each question's prompt is [p; c_b; x_i].  Rows
    of p are causal over p, context rows see all of p, question rows all of p
    and c_b; every row is checked against the fp64 oracle, and every pool row
    outside the instructions and contexts keeps its sentinel."""
    name, wid, dtype, hq, hkv, d, B, ctx, qs, ql, cpi, lp = case
    log(f"case: two-level prefill {name} standard={standard} tile_rows={rows}")
    wl = W.custom_workload(wid=wid, dtype=dtype, num_prompts=B, hq=hq, hkv=hkv,
                           head_dim=d, ctx_len=ctx, questions=qs, question_tokens=0, seg_len=ql,
                           value_std=0.5 if dtype == "bf16" else 1.0)
    st = W.make_structure(wl)
    kv = W.layer_kv(st)
    pq = W.prefill_queries(st)
    ins = W.instructions(st, cpi, lp)
    iq = W.instruction_queries(st, ins)
    cap = max(8, int(st.seg_len0.max()) if st.num_questions else 8)
    db = DecodeBatch(st.ctx_len.tolist(), st.q_count.tolist(), wl.hq, wl.hkv, wl.head_dim, wl.dtype, cap,
                     rope_base=wl.rope_base, instr_len=ins.lp.tolist(), instr_prompt_start=ins.prompt_start.tolist(),
                     tile_rows=rows)
    db.load_instructions(0, ins.k, ins.v)
    db.load_context(0, kv.ctx_k, kv.ctx_v)
    db.load_segments(0, kv.seg_k, kv.seg_v, st.seg_len0)
    q_ctx, q_seg = db.pack_prefill_queries(pq.ctx_q, pq.seg_q, st.seg_len0, instr_q=iq)
    oc, os_ = db.prefill_outputs(fill=SENTINEL)
    per_prompt = [int(st.seg_len0[st.q_start[b]:st.q_start[b + 1]].sum()) for b in range(wl.num_prompts)]
    db.prefill(0, q_ctx, q_seg, oc, os_, max(per_prompt + [0]), standard=standard)
    torch.cuda.synchronize()
    oc_h, os_h = oc.cpu().numpy(), os_.cpu().numpy()
    S = len(ins.lp)
    g_ctx = np.concatenate([oc_h[db.ctx_off[b]: db.ctx_off[b] + st.ctx_len[b]] for b in range(wl.num_prompts)])
    g_ins = np.concatenate([oc_h[db.instr_off[s]: db.instr_off[s] + ins.lp[s]] for s in range(S)])
    g_seg = (np.concatenate([os_h[i, : st.seg_len0[i]] for i in range(st.num_questions)])
             if st.num_questions else np.zeros((0, wl.hq, wl.head_dim)))
    r_ctx, r_seg, r_ins = P.prefill_standard(kv.ctx_k, kv.ctx_v, pq.ctx_q, st.ctx_start, st.q_start, kv.seg_k,
                                             kv.seg_v, pq.seg_q, st.seg_start, wl.rope_base,
                                             instr=(ins.prompt_start, ins.tok_start, ins.k, ins.v, iq))
    written = np.zeros(db.pool, bool)
    for b in range(wl.num_prompts):
        if standard and st.q_count[b] == 0:
            # no question's prompt holds this context: its rows stay untouched
            rows = slice(st.ctx_start[b], st.ctx_start[b + 1])
            assert (g_ctx[rows] == SENTINEL).all()
            r_ctx[rows] = np.nan
            continue
        written[db.ctx_off[b]: db.ctx_off[b] + st.ctx_len[b]] = True
    for s in range(S):
        nq = int(st.q_start[ins.prompt_start[s + 1]] - st.q_start[ins.prompt_start[s]])
        rows = slice(ins.tok_start[s], ins.tok_start[s + 1])
        if standard and nq == 0:
            assert (g_ins[rows] == SENTINEL).all()
            r_ins[rows] = np.nan
            continue
        written[db.instr_off[s]: db.instr_off[s] + ins.lp[s]] = True
    e_ctx, e_seg, e_ins = max_err(g_ctx, r_ctx), max_err(g_seg, r_seg), max_err(g_ins, r_ins)
    log(f"  instr rows {len(g_ins)} err {e_ins:.3e}; ctx rows {len(g_ctx)} err {e_ctx:.3e}; "
        f"question rows {len(g_seg)} err {e_seg:.3e}")
    assert max(e_ctx, e_seg, e_ins) <= tol(dtype)
    assert (oc_h[~written] == SENTINEL).all()
    for i in range(st.num_questions):
        assert (os_h[i, st.seg_len0[i]:] == SENTINEL).all()
    assert db.err_flag() == 0


@pytest.mark.parametrize("rows", [0, 256])
@pytest.mark.parametrize("standard", [False, True])
def test_prefill_maximum_questions_and_group(standard, rows):
    """1024 questions of 0..3 tokens in one prompt (the prefill's question
    list at its length) with G = 16, bf16 at D = 128: sampled rows against the
    oracle, the rest finite, sentinels past every question's tokens."""
    log(f"case: prefill 1024 questions, G=16, standard={standard}, tile_rows={rows}")
    wl = W.custom_workload(wid=470, dtype="bf16", num_prompts=1, hq=32, hkv=2, head_dim=128, ctx_len=(300, 300),
                           questions=(1024, 1024), question_tokens=0, seg_len=(0, 3), value_std=0.5)
    rng = np.random.default_rng(11)
    ctx_rows = sorted(set([0, 31, 32, 299] + rng.integers(0, 300, 8).tolist()))
    st0 = W.make_structure(wl)
    nseg = int(st0.seg_start[-1])
    seg_rows = sorted(set([0, nseg - 1] + rng.integers(0, nseg, 60).tolist()))
    st, g_ctx, g_seg, r_ctx, r_seg, db, oc_h, os_h = prefill_case(wl, standard=standard, ctx_rows=ctx_rows,
                                                                 seg_rows=seg_rows, tile_rows=rows)
    assert int((st.seg_len0 == 0).sum()) > 0
    e_ctx = max_err(g_ctx[ctx_rows], r_ctx[ctx_rows])
    e_seg = max_err(g_seg[seg_rows], r_seg[seg_rows])
    log(f"  sampled ctx max err {e_ctx:.3e}, question max err {e_seg:.3e} ({nseg} question tokens)")
    assert e_ctx <= 2e-2 and e_seg <= 2e-2
    assert np.isfinite(g_ctx).all() and np.isfinite(g_seg).all()
    check_unwritten(st, db, oc_h, os_h, standard)
    assert db.err_flag() == 0
