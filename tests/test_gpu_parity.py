"""GPU parity: the HIP path through the C ABI against the fp64 oracle.

Tolerances: max |gpu - oracle| <= 1e-5 for fp32 workloads, <= 2e-2 for bf16
operands with fp32 accumulation, on out and on lse.
"""
import numpy as np
import pytest
import torch

import workload as W
from oracle import ippd as O
from tests.gpu_harness import (load_layer, log, make_batch, max_err, oracle_steps,
                               run_gpu)

pytestmark = pytest.mark.gpu

TOL = {"f32": 1e-5, "bf16": 2e-2}


def check(st, gpu, ref, steps, label, qsel=None):
    tol = TOL[st.wl.dtype]
    for t in steps:
        ro, rl = ref[t]
        go, gl = gpu.out[t], gpu.lse[t]
        if qsel is not None:
            idx = [i for i in qsel[t] if st.active(t)[i]]
            ro, rl, go, gl = ro[idx], rl[idx], go[idx], gl[idx]
        eo, el = max_err(go, ro), max_err(gl, rl)
        log(f"{label} step {t}: max|out err| {eo:.3e}  max|lse err| {el:.3e}  (tol {tol})")
        assert eo <= tol and el <= tol, (label, t, eo, el)


# ------------------------------------------------------------------ tiny fp32

def test_tiny_f32_full():
    log("case: tiny fp32 workload, 1 step")
    wl = W.workload(1)
    st = W.make_structure(wl)
    kv = W.layer_kv(st)
    gpu = run_gpu(st, [0], [0], kv=kv)
    ref = oracle_steps(st, kv, [0], [0])
    assert gpu.err == 0
    check(st, gpu, ref, [0], "tiny-f32")

    # rotated query and the appended key/value at virtual position Lc + s_i
    si = W.step_inputs(st, 0)
    pos = st.ctx_len[0] + st.seg_len0
    q_ref = O.rope(si.q_new, pos[:, None], wl.rope_base)
    np.testing.assert_allclose(gpu.q_rot[0], q_ref, atol=2e-6, rtol=0)
    db = gpu.batch
    seg_k = db.seg_k[0].float().cpu().numpy()
    seg_vt = db.seg_values(0).float().cpu().numpy()
    for i in range(st.num_questions):
        s = st.seg_len0[i]
        k_ref = O.rope(si.k_new[i], pos[i], wl.rope_base)
        np.testing.assert_allclose(seg_k[i, :, s], k_ref, atol=2e-6, rtol=0)
        np.testing.assert_array_equal(seg_vt[i, :, :, s], si.v_new[i])
    assert db.seg_len[0][: st.num_questions].cpu().numpy().tolist() == (st.seg_len0 + 1).tolist()
    # context cache rotated at positions 0..Lc-1, values transposed
    ck = db.ctx_k[0].float().cpu().numpy()
    k_ctx_ref = O.rope(kv.ctx_k.transpose(1, 0, 2), np.arange(256)[None, :], wl.rope_base)
    np.testing.assert_allclose(ck[:, :256], k_ctx_ref, atol=2e-6, rtol=0)
    np.testing.assert_array_equal(db.ctx_values(0).float().cpu().numpy()[:, :, :256],
                                  kv.ctx_v.transpose(1, 2, 0))


# ------------------------------------------------------------- small ragged

def ragged_workload(dtype, d=64, hq=8, hkv=2, steps=3, seed_id=200):
    return W.custom_workload(wid=seed_id, dtype=dtype, num_prompts=3, hq=hq, hkv=hkv, head_dim=d,
                             ctx_len=(40, 200), questions=(1, 6), question_tokens=0,
                             seg_len=(1, 40), steps=steps, stop=(1, steps),
                             value_std=1.0 if dtype == "f32" else 0.5)


@pytest.mark.parametrize("fused", [False, True])
@pytest.mark.parametrize("dtype,d,chunk,rows", [("f32", 64, 0, 0), ("f32", 128, 32, 16), ("bf16", 128, 0, 0),
                                                ("bf16", 128, 64, 32), ("bf16", 64, 32, 64),
                                                ("bf16", 128, 96, 16), ("bf16", 128, 160, 128),
                                                ("f32", 64, 64, 128)])
def test_small_ragged(dtype, d, chunk, rows, fused):
    log(f"case: small ragged dtype={dtype} D={d} chunk={chunk} tile_rows={rows} fused={fused}")
    st = W.make_structure(ragged_workload(dtype, d))
    kv = W.layer_kv(st)
    steps = list(range(st.wl.steps))
    gpu = run_gpu(st, steps, steps, chunk_tokens=chunk, kv=kv, fused=fused, tile_rows=rows)
    ref = oracle_steps(st, kv, steps, steps)
    assert gpu.err == 0
    check(st, gpu, ref, steps, f"ragged-{dtype}-{d}-{chunk}-{rows}-{'fused' if fused else 'sep'}")
    np.testing.assert_array_equal(gpu.batch.seg_len[0][: st.num_questions].cpu().numpy(),
                                  st.seg_len_at(st.wl.steps))


@pytest.mark.parametrize("fused", [False, True])
@pytest.mark.parametrize("ctx,chunk", [(37, 0), (200, 0), (200, 64), (200, 96), (300, 96)])
def test_eight_wave_units_odd_and_short_tile_counts(ctx, chunk, fused):
    """Prompts of one context length with 32 questions of G = 4 heads: the
    planner's eight single-block waves per 128-row unit, whose loop folds two
    tiles per barrier.  Context lengths and chunk sizes give units of 1, 2, 3,
    7 and 10 tiles (odd counts fold their last tile alone, units shorter than
    the ring start with a partial prologue), partial last tiles, and a second
    step after some questions stopped."""
    log(f"case: eight-wave units ctx={ctx} chunk={chunk} fused={fused}")
    wl = W.custom_workload(wid=280, dtype="bf16", num_prompts=2, hq=32, hkv=8, head_dim=128,
                           ctx_len=(ctx, ctx), questions=(32, 32), question_tokens=0, seg_len=(1, 40),
                           steps=2, stop=(1, 2))
    st = W.make_structure(wl)
    kv = W.layer_kv(st)
    gpu = run_gpu(st, [0, 1], [0, 1], chunk_tokens=chunk, kv=kv, fused=fused)
    assert gpu.err == 0
    ref = oracle_steps(st, kv, [0, 1], [0, 1])
    check(st, gpu, ref, [0, 1], f"eight-wave-{ctx}-{chunk}-{'fused' if fused else 'sep'}")


@pytest.mark.parametrize("mode", ["fused", "separate", "standard"])
def test_more_than_64_prompts(mode):
    """80 ragged prompts: the prompt lookups take their second window of 64
    (segment units, standard context units, the append kernel), and the
    pool-sized chunk splits the longer contexts into equal chunks.  Every
    question against the oracle over two steps with stops after the first."""
    log(f"case: 80 prompts, mode={mode}")
    wl = W.custom_workload(wid=270, dtype="bf16", num_prompts=80, hq=8, hkv=2, head_dim=128,
                           ctx_len=(24, 400), questions=(1, 3), seg_len=(1, 30), steps=2, stop=(1, 2))
    st = W.make_structure(wl)
    kv = W.layer_kv(st)
    gpu = run_gpu(st, [0, 1], [0, 1], kv=kv, fused=mode != "separate", standard=mode == "standard")
    assert gpu.err == 0
    ref = oracle_steps(st, kv, [0, 1], [0, 1])
    check(st, gpu, ref, [0, 1], f"80-prompts-{mode}")
    if mode != "standard":
        np.testing.assert_array_equal(gpu.batch.seg_len[0][: st.num_questions].cpu().numpy(), st.seg_len_at(2))


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_fused_step_equals_separate_calls(dtype):
    """ippd_decode_step == ippd_append_kv + ippd_decode_attention (same rotation, same
    partial regrouping), and its q_rot output equals the append's."""
    log(f"case: fused vs separate dtype={dtype}")
    st = W.make_structure(ragged_workload(dtype, 128, steps=3))
    kv = W.layer_kv(st)
    steps = list(range(3))
    a = run_gpu(st, steps, steps, kv=kv, fused=False)
    b = run_gpu(st, steps, steps, kv=kv, fused=True)
    for t in steps:
        act = st.active(t)
        np.testing.assert_array_equal(a.out[t][act], b.out[t][act])
        np.testing.assert_array_equal(a.q_rot[t][act], b.q_rot[t][act])
    ka, kb = a.batch.seg_k[0].float().cpu().numpy(), b.batch.seg_k[0].float().cpu().numpy()
    va, vb = a.batch.seg_values(0).float().cpu().numpy(), b.batch.seg_values(0).float().cpu().numpy()
    for i, n in enumerate(st.seg_len_at(3)):           # filled slots only
        np.testing.assert_array_equal(ka[i, :, :n], kb[i, :, :n])
        np.testing.assert_array_equal(va[i, :, :, :n], vb[i, :, :, :n])


@pytest.mark.parametrize("fused", [False, True])
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_standard_baseline_matches_oracle(dtype, fused):
    log(f"case: standard baseline dtype={dtype} fused={fused}")
    st = W.make_structure(ragged_workload(dtype, 128))
    kv = W.layer_kv(st)
    steps = list(range(st.wl.steps))
    gpu = run_gpu(st, steps, steps, standard=True, kv=kv, fused=fused)
    ref = oracle_steps(st, kv, steps, steps)
    check(st, gpu, ref, steps, f"standard-{dtype}-{'fused' if fused else 'sep'}")


@pytest.mark.parametrize("mode,fused", [("ippd", False), ("ippd", True), ("standard", False), ("standard", True),
                                        ("dense", False)])
def test_workspace_needs_no_initialisation(mode, fused):
    """Every partial state a call reads is written earlier in the same call:
    with the workspace refilled with 0xFF bytes (NaN) before every call, each
    decode mode gives the oracle's results."""
    log(f"case: NaN-filled workspace mode={mode} fused={fused}")
    st = W.make_structure(ragged_workload("bf16", 128, steps=3))
    kv = W.layer_kv(st)
    db = make_batch(st, chunk_tokens=64)
    load_layer(db, st, 0, kv)
    if mode == "dense":
        db.ws_dense = torch.empty(db.ws_dense_bytes, dtype=torch.uint8, device=db.device)
    ws = {"ippd": db.ws_ippd, "standard": db.ws_std, "dense": db.ws_dense if mode == "dense" else None}[mode]
    steps = list(range(3))
    ref = oracle_steps(st, kv, steps, steps)
    for t in steps:
        si = W.step_inputs(st, t)
        db.set_active(si.active)
        q, k, v = db.to_dev(si.q_new), db.to_dev(si.k_new), db.to_dev(si.v_new)
        ws.fill_(0xFF)
        if fused:
            db.decode_step(0, q, k, v, standard=mode == "standard")
        else:
            db.append(0, q, k, v)
            db.decode(0, standard=mode == "standard", dense=mode == "dense")
        torch.cuda.synchronize()
        act = st.active(t)
        eo = max_err(db.out[: st.num_questions].cpu().numpy()[act], ref[t][0][act])
        el = max_err(db.lse[: st.num_questions].cpu().numpy()[act], ref[t][1][act])
        log(f"nan-workspace-{mode}-{'fused' if fused else 'sep'} step {t}: out {eo:.3e} lse {el:.3e}")
        assert eo <= TOL["bf16"] and el <= TOL["bf16"], (mode, t, eo, el)
    assert db.err_flag() == 0


def test_inactive_rows_untouched_and_not_appended():
    log("case: inactive rows keep the sentinel, their segments do not grow")
    st = W.make_structure(ragged_workload("bf16", 128, steps=4))
    kv = W.layer_kv(st)
    steps = list(range(4))
    gpu = run_gpu(st, steps, steps, sentinel=-777.0, kv=kv, fused=True)
    for t in steps:
        dead = ~st.active(t)
        assert np.all(gpu.out[t][dead] == -777.0) and np.all(gpu.lse[t][dead] == -777.0)
        assert not np.any(gpu.out[t][~dead] == -777.0)
    got = gpu.batch.seg_len[0][: st.num_questions].cpu().numpy()
    np.testing.assert_array_equal(got, st.seg_len_at(4))


def test_split_count_and_batch_independence():
    """Chunking regroups exact sums (results agree across chunk sizes); a prompt's
    output does not depend on the other prompts of the batch (Sec. 4.4)."""
    log("case: split-count / batch independence")
    wl = W.custom_workload(wid=210, dtype="bf16", num_prompts=3, hq=32, hkv=8, head_dim=128,
                           ctx_len=(300, 900), questions=(3, 9), seg_len=(5, 60), steps=1)
    st = W.make_structure(wl)
    kv = W.layer_kv(st)
    outs = {}
    for ch in (32, 96, 256, 1024):
        outs[ch] = run_gpu(st, [0], [0], chunk_tokens=ch, kv=kv).out[0]
    ref = oracle_steps(st, kv, [0], [0])
    for ch, o in outs.items():
        e = max_err(o, ref[0][0])
        log(f"chunk {ch}: max err {e:.3e}")
        assert e <= TOL["bf16"]
        assert np.max(np.abs(o - outs[32])) <= 2e-3
    # prompt 1 alone
    b = 1
    st1 = W.Structure(wl, st.ctx_len[b:b + 1], st.q_count[b:b + 1],
                      st.seg_len0[st.q_start[b]:st.q_start[b + 1]], st.stop[st.q_start[b]:st.q_start[b + 1]])
    kv1 = W.LayerKV(kv.ctx_k[st.ctx_start[b]:st.ctx_start[b + 1]], kv.ctx_v[st.ctx_start[b]:st.ctx_start[b + 1]],
                    kv.seg_k[st.seg_start[st.q_start[b]]:st.seg_start[st.q_start[b + 1]]],
                    kv.seg_v[st.seg_start[st.q_start[b]]:st.seg_start[st.q_start[b + 1]]])
    db = make_batch(st1, chunk_tokens=96, max_questions=int(st.q_count.max()))
    load_layer(db, st1, 0, kv1)
    si = W.step_inputs(st, 0)
    sl = slice(st.q_start[b], st.q_start[b + 1])
    db.set_active(si.active[sl])
    db.append(0, db.to_dev(si.q_new[sl]), db.to_dev(si.k_new[sl]), db.to_dev(si.v_new[sl]))
    db.decode(0)
    alone = db.out[: st1.num_questions].cpu().numpy()
    np.testing.assert_array_equal(alone, outs[96][sl])


def test_empty_context_and_many_questions():
    log("case: a prompt with an empty context and a prompt with 300 questions")
    wl = W.custom_workload(wid=220, dtype="bf16", num_prompts=2, hq=8, hkv=2, head_dim=128,
                           steps=1)
    rng = np.random.default_rng(5)
    q_count = np.array([3, 300])
    st = W.Structure(wl, np.array([0, 150]), q_count, rng.integers(1, 20, size=303),
                     np.full(303, 1))
    kv = W.layer_kv(st)
    gpu = run_gpu(st, [0], [0], kv=kv)
    assert gpu.err == 0
    sel = {0: list(range(0, 303, 7)) + [0, 1, 2]}
    ref = oracle_steps(st, kv, [0], [0], questions=sel)
    check(st, gpu, ref, [0], "empty-ctx/300q", qsel=sel)


@pytest.mark.parametrize("fused", [False, True])
def test_group_of_three_heads(fused):
    """G = 3 query heads per kv head: a 16-row tile boundary falls inside a question
    (rows per context unit 16..256; 128 and 256 put two 16-row blocks on a wave)."""
    log(f"case: G=3 (Hq 6, Hkv 2) fused={fused}")
    wl = W.custom_workload(wid=240, dtype="bf16", num_prompts=2, hq=6, hkv=2, head_dim=128,
                           ctx_len=(90, 300), questions=(7, 13), seg_len=(2, 30), steps=2,
                           value_std=0.5)
    st = W.make_structure(wl)
    kv = W.layer_kv(st)
    for rows in (16, 32, 64, 128, 256):
        gpu = run_gpu(st, [0, 1], [0, 1], kv=kv, fused=fused, tile_rows=rows, chunk_tokens=64)
        ref = oracle_steps(st, kv, [0, 1], [0, 1])
        assert gpu.err == 0
        check(st, gpu, ref, [0, 1], f"G3-rows{rows}")


def test_rope_base_500000_f32():
    log("case: rope base 5e5, fp32")
    wl = W.custom_workload(wid=230, dtype="f32", num_prompts=2, hq=4, hkv=4, head_dim=64,
                           ctx_len=(500, 700), questions=(2, 3), seg_len=(3, 9), steps=2,
                           rope_base=500000.0, value_std=1.0)
    st = W.make_structure(wl)
    kv = W.layer_kv(st)
    gpu = run_gpu(st, [0, 1], [0, 1], kv=kv)
    ref = oracle_steps(st, kv, [0, 1], [0, 1])
    check(st, gpu, ref, [0, 1], "base5e5")


def test_all_inactive_step_is_a_noop():
    log("case: every question stopped")
    st = W.make_structure(ragged_workload("bf16", 128, steps=2))
    db = make_batch(st)
    load_layer(db, st, 0, W.layer_kv(st))
    si = W.step_inputs(st, 0)
    db.set_active(np.zeros(st.num_questions, bool))
    db.out.fill_(3.0)
    before = db.seg_len[0].clone()
    db.append(0, db.to_dev(si.q_new), db.to_dev(si.k_new), db.to_dev(si.v_new))
    db.decode(0)
    torch.cuda.synchronize()
    assert torch.all(db.out == 3.0)
    assert torch.equal(db.seg_len[0], before)
    assert db.err_flag() == 0


@pytest.mark.parametrize("mode", ["ippd", "standard", "dense"])
def test_device_side_flags(mode):
    """A full segment and a broken prompt layout raise their flags; the
    questions of the broken prompt get no output row (their rows keep the
    sentinel) and every other question is still served."""
    log(f"case: segment overflow and bad layout raise flags, affected rows skipped ({mode})")
    st = W.make_structure(ragged_workload("bf16", 64, steps=1))
    db = make_batch(st, extra_cap=0)
    load_layer(db, st, 0, W.layer_kv(st))
    seg0 = db.seg_len[0].clone()
    # fill every segment to capacity, then append: overflow flag, seg_len unchanged
    db.seg_len[0][: st.num_questions] = db.seg_cap
    si = W.step_inputs(st, 0)
    db.set_active(np.ones(st.num_questions, bool))
    db.append(0, db.to_dev(si.q_new), db.to_dev(si.k_new), db.to_dev(si.v_new))
    torch.cuda.synchronize()
    assert db.err_flag() & 1
    assert int(db.seg_len[0][0]) == db.seg_cap
    # misaligned context offset of prompt 0: attention skips its questions and flags it
    db.seg_len[0].copy_(seg0)
    db.append(0, db.to_dev(si.q_new), db.to_dev(si.k_new), db.to_dev(si.v_new))
    db.d_err.zero_()
    db.d_ctx_off[0] = 3
    db.out.fill_(-777.0)
    if mode == "dense":
        db.ws_dense = torch.empty(db.ws_dense_bytes, dtype=torch.uint8, device=db.device)
        db.ws_dense.fill_(0xFF)
    db.decode(0, standard=mode == "standard", dense=mode == "dense")
    torch.cuda.synchronize()
    assert db.err_flag() & 2
    out = db.out[: st.num_questions].cpu().numpy()
    q0, q1 = int(st.q_start[0]), int(st.q_start[1])
    assert np.all(out[q0:q1] == -777.0), "rows of the broken prompt were written"
    assert np.all(np.isfinite(out[q1:])) and not np.any(out[q1:] == -777.0)


# -------------------------------------------------------- full-size workloads

def test_llama3_8b_lc4096_n16_64_steps():
    log("case: workload 2 (Lc 4096, N 16, 64 steps), sampled steps vs oracle")
    st = W.make_structure(W.workload(2))
    kv = W.layer_kv(st)
    steps = list(range(64))
    rec = [0, 1, 32, 63]
    gpu = run_gpu(st, steps, rec, kv=kv, fused=True)
    assert gpu.err == 0
    ref = oracle_steps(st, kv, steps, rec)
    check(st, gpu, ref, rec, "wl2")
    std = run_gpu(st, [0], [0], standard=True, kv=kv, fused=True)
    check(st, std, {0: ref[0]}, [0], "wl2-standard")
    sep = run_gpu(st, [0], [0], kv=kv, fused=False)
    check(st, sep, {0: ref[0]}, [0], "wl2-separate")


def test_ragged_b32_sampled():
    log("case: workload 3 (B 32 ragged, 32 steps), sampled questions vs oracle")
    st = W.make_structure(W.workload(3))
    kv = W.layer_kv(st)
    steps = list(range(32))
    rec = [0, 31]
    rng = np.random.default_rng(0)
    sel = {t: sorted(rng.choice(st.num_questions, 20, replace=False).tolist()) for t in rec}
    gpu = run_gpu(st, steps, rec, kv=kv, fused=True)
    assert gpu.err == 0
    ref = oracle_steps(st, kv, steps, rec, questions=sel)
    check(st, gpu, ref, rec, "wl3", qsel=sel)


def test_long_context_sampled():
    """Workload 4, the only one with 256-row units: every question at the last
    step, sampled questions at the first."""
    log("case: workload 4 (Lc 32768, N 64, 32 steps), all 64 questions at step 31 vs oracle")
    st = W.make_structure(W.workload(4))
    kv = W.layer_kv(st)
    steps = list(range(32))
    rec = [0, 31]
    sel = {0: [0, 17, 40, 63], 31: list(range(64))}
    gpu = run_gpu(st, steps, rec, kv=kv, fused=True)
    assert gpu.err == 0
    ref = oracle_steps(st, kv, steps, rec, questions=sel)
    check(st, gpu, ref, rec, "wl4", qsel=sel)


@pytest.mark.parametrize("layer", [0, 31])
def test_32layer_sampled(layer):
    log(f"case: workload 5 layer {layer} (B 8, Lc 8192, 128 steps, shrinking active set)")
    st = W.make_structure(W.workload(5))
    kv = W.layer_kv(st, layer)
    steps = list(range(128))
    rec = [0, 15, 64, 127]
    rng = np.random.default_rng(layer)
    sel = {t: sorted(rng.choice(st.num_questions, 8, replace=False).tolist()) for t in rec}
    gpu = run_gpu(st, steps, rec, layer=layer, kv=kv, fused=True)
    assert gpu.err == 0
    ref = oracle_steps(st, kv, steps, rec, layer=layer, questions=sel)
    check(st, gpu, ref, rec, f"wl5-L{layer}", qsel=sel)


def test_32layer_late_steps_every_active_question():
    """Workload 5 late in its 128 steps, where most questions have stopped and
    the context units serve only the compacted active rows: every question
    still active at steps 96 and 127 against the oracle, and the stopped
    questions' rows left as they were."""
    st = W.make_structure(W.workload(5))
    kv = W.layer_kv(st, 0)
    rec = [96, 127]
    act = {t: np.flatnonzero(st.active(t)).tolist() for t in rec}
    log(f"case: workload 5 late steps, active questions {[len(a) for a in act.values()]} of {st.num_questions}")
    assert 0 < len(act[127]) < len(act[96]) < st.num_questions // 2
    gpu = run_gpu(st, range(128), rec, kv=kv, fused=True, sentinel=-777.0)
    assert gpu.err == 0
    for t in rec:
        stopped = ~st.active(t)
        assert np.all(gpu.out[t][stopped] == -777.0) and np.all(gpu.lse[t][stopped] == -777.0)
    ref = oracle_steps(st, kv, range(128), rec, questions=act)
    check(st, gpu, ref, rec, "wl5-late", qsel=act)


@pytest.mark.parametrize("mode", ["separate", "fused", "standard"])
def test_maximum_questions_and_group(mode):
    """The documented maxima together: 1024 questions in one prompt (the length
    of a prompt's question list) and G = 16 query heads per kv head (a question
    fills one 16-row MFMA block), bf16 at D = 128, over two steps with about a
    third of the questions stopping after the first; empty segments included.
    Sampled questions against the oracle, which computes them one by one."""
    log(f"case: 1024 questions in one prompt, G=16, mode={mode}")
    wl = W.custom_workload(wid=260, dtype="bf16", num_prompts=2, hq=32, hkv=2, head_dim=128, steps=2,
                           value_std=0.5)
    rng = np.random.default_rng(9)
    nt = 1025
    st = W.Structure(wl, np.array([600, 130]), np.array([1024, 1]), rng.integers(0, 24, size=nt),
                     rng.choice([1, 2], size=nt, p=[1 / 3, 2 / 3]))
    kv = W.layer_kv(st)
    gpu = run_gpu(st, [0, 1], [0, 1], kv=kv, fused=mode == "fused", standard=mode == "standard")
    assert gpu.err == 0
    picks = sorted(set([0, 1, 15, 16, 511, 512, 1022, 1023, 1024] + rng.integers(0, nt, 40).tolist()))
    sel = {0: picks, 1: picks}
    ref = oracle_steps(st, kv, [0, 1], [0, 1], questions=sel)
    check(st, gpu, ref, [0, 1], f"1024q-G16-{mode}", qsel=sel)
