"""Pins of the fp64 oracle against what the paper and mathematics fix.

None of these compares the oracle with itself: each pin is a closed form, a
library routine, a 50-digit brute force written in a different form, a
hand-derived fixture, or an invariant the paper states.  A planted-mistake
section at the end shows that plausible slips in the oracle fail a pin.
"""
import math
import os

import mpmath
import numpy as np
import pytest
import torch

import oracle
from oracle import ippd as O
import workload as W

GOLDEN = os.path.join(os.path.dirname(__file__), "golden")


def rng(seed):
    return np.random.default_rng(seed)


# ---------------------------------------------------------------- rotary ---

def rope_complex(x, pos, base):
    """Rotary embedding written as complex multiplication z_j * e^{i pos theta_j},
    with z_j = x_j + i x_{j+D/2} (an independent form of the rotate-half map)."""
    d = x.shape[-1]
    h = d // 2
    theta = np.array([base ** (-(2.0 * j) / d) for j in range(h)])
    z = x[..., :h] + 1j * x[..., h:]
    z = z * np.exp(1j * np.asarray(pos, float)[..., None] * theta)
    return np.concatenate([z.real, z.imag], axis=-1)


def test_rope_matches_complex_form():
    x = rng(1).standard_normal((5, 7, 64))
    pos = rng(2).integers(0, 40000, size=(5, 7))
    for base in (10000.0, 500000.0):
        # fp64 angles up to 4e4 rad carry ~pos * 1e-16 absolute error in either form
        np.testing.assert_allclose(O.rope(x, pos, base), rope_complex(x, pos, base),
                                   rtol=0, atol=1e-10)


def test_rope_pairing_closed_form():
    # D = 4, theta = (1, base^-1/2): unit vector e_0 at position m -> (cos m, 0, sin m, 0),
    # e_1 -> (0, cos m t1, 0, sin m t1).  Pins the (j, j + D/2) pairing and the sign.
    base, m = 100.0, 3
    t1 = base ** -0.5
    np.testing.assert_allclose(O.rope(np.array([1., 0, 0, 0]), m, base),
                               [math.cos(m), 0, math.sin(m), 0], atol=1e-15)
    np.testing.assert_allclose(O.rope(np.array([0., 1, 0, 0]), m, base),
                               [0, math.cos(m * t1), 0, math.sin(m * t1)], atol=1e-15)
    np.testing.assert_allclose(O.rope(np.array([0., 0, 1, 0]), m, base),
                               [-math.sin(m), 0, math.cos(m), 0], atol=1e-15)


def test_rope_group_properties():
    x = rng(3).standard_normal((9, 128))
    np.testing.assert_array_equal(O.rope(x, 0, 10000.0), x)                   # R(0) = I
    r = O.rope(x, 12345, 10000.0)
    np.testing.assert_allclose(np.linalg.norm(r, axis=-1), np.linalg.norm(x, axis=-1),
                               rtol=1e-13)                                      # isometry
    np.testing.assert_allclose(O.rope(O.rope(x, 17, 1e4), 29, 1e4), O.rope(x, 46, 1e4),
                               atol=1e-12)                                      # R(a)R(b)=R(a+b)


def test_rope_relative_position():
    # <R(m) q, R(n) k> depends only on m - n: shifting both positions leaves logits unchanged.
    q, k = rng(4).standard_normal((2, 128))
    a = O.rope(q, 300, 1e4) @ O.rope(k, 100, 1e4)
    b = O.rope(q, 4300, 1e4) @ O.rope(k, 4100, 1e4)
    assert abs(a - b) < 1e-10


def test_rope_d2_logit_closed_form():
    # D = 2, theta_0 = 1: logit = |q||k| cos(phi_q - phi_k + (m_q - m_k)) / sqrt(2).
    q, k = np.array([0.3, -1.1]), np.array([2.0, 0.5])
    mq, mk = 7, 3
    got = O.rope(q, mq, 1e4) @ O.rope(k, mk, 1e4) / math.sqrt(2)
    phq, phk = math.atan2(q[1], q[0]), math.atan2(k[1], k[0])
    want = np.linalg.norm(q) * np.linalg.norm(k) * math.cos(phq - phk + (mq - mk)) / math.sqrt(2)
    assert abs(got - want) < 1e-14


# ------------------------------------------------------------- attention ---

def test_attend_closed_forms():
    r = rng(5)
    K = r.standard_normal((11, 16))
    V = r.standard_normal((11, 16))
    out, lse = O.attend(np.zeros(16), K, V, 0.25)
    np.testing.assert_allclose(out, V.mean(0), atol=1e-14)                     # q = 0 -> mean V
    assert abs(lse - math.log(11)) < 1e-14                                     # lse = ln n
    const = np.tile(r.standard_normal(16), (11, 1))
    out, _ = O.attend(r.standard_normal(16), K, const, 0.25)
    np.testing.assert_allclose(out, const[0], atol=1e-14)                      # constant V
    q = np.zeros(16); q[0] = 1.0
    Kb = np.zeros((11, 16)); Kb[4, 0] = 1e4
    out, _ = O.attend(q, Kb, V, 1.0)
    np.testing.assert_allclose(out, V[4], atol=1e-12)                          # one dominant key


def _small_case(seed, B=2, hq=4, hkv=2, d=16, lc=(5, 9), nq=(2, 3), sl=(1, 4), lp=0):
    r = rng(seed)
    ctx_len = r.integers(lc[0], lc[1] + 1, size=B)
    q_count = r.integers(nq[0], nq[1] + 1, size=B)
    q_start = np.concatenate([[0], np.cumsum(q_count)])
    ctx_start = np.concatenate([[0], np.cumsum(ctx_len)])
    nt = int(q_start[-1])
    seg_len = r.integers(sl[0], sl[1] + 1, size=nt)
    ck = r.standard_normal((ctx_start[-1], hkv, d))
    cv = r.standard_normal((ctx_start[-1], hkv, d))
    sk = [r.standard_normal((s, hkv, d)) for s in seg_len]
    sv = [r.standard_normal((s, hkv, d)) for s in seg_len]
    q = r.standard_normal((nt, hq, d))
    k = r.standard_normal((nt, hkv, d))
    v = r.standard_normal((nt, hkv, d))
    ik = r.standard_normal((lp, hkv, d)) if lp else None
    iv = r.standard_normal((lp, hkv, d)) if lp else None
    return dict(ck=ck, cv=cv, ctx_start=ctx_start, q_start=q_start, sk=sk, sv=sv,
                q=q, k=k, v=v, ik=ik, iv=iv, seg_len=seg_len)


def test_single_question_is_causal_attention_sdpa():
    """N = 1 reduces to plain causal attention: last row of torch SDPA (fp64, GQA)."""
    r = rng(6)
    hq, hkv, d, lc, s, base = 8, 2, 32, 13, 5, 10000.0
    ck, cv = r.standard_normal((2, lc, hkv, d))
    sk, sv = r.standard_normal((2, s, hkv, d))
    qn = r.standard_normal((hq, d))
    kn, vn = r.standard_normal((2, hkv, d))
    out, lse = O.standard_prompting_question(ck, cv, sk, sv, qn, kn, vn, base)

    n = lc + s + 1
    Kraw = np.concatenate([ck, sk, kn[None]])          # [n, hkv, d]
    Vall = np.concatenate([cv, sv, vn[None]])
    Qraw = r.standard_normal((n, hq, d))
    Qraw[-1] = qn                                      # earlier rows: arbitrary queries
    Kr = np.stack([rope_complex(Kraw[t], t, base) for t in range(n)])
    Qr = np.stack([rope_complex(Qraw[t], t, base) for t in range(n)])
    qt = torch.from_numpy(Qr).permute(1, 0, 2)[None]   # [1, hq, n, d]
    kt = torch.from_numpy(Kr).permute(1, 0, 2)[None]
    vt = torch.from_numpy(Vall).permute(1, 0, 2)[None]
    ref = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, is_causal=True,
                                                           enable_gqa=True)
    np.testing.assert_allclose(out, ref[0, :, -1].numpy(), atol=1e-12)
    # lse against a logsumexp over the same logits computed by torch
    logits = torch.einsum("hd,hnd->hn", qt[0, :, -1], kt[0].repeat_interleave(hq // hkv, 0))
    np.testing.assert_allclose(lse, torch.logsumexp(logits / math.sqrt(d), -1).numpy(),
                               atol=1e-12)


@pytest.mark.parametrize("seed,lp", [(10, 0), (11, 3), (12, 1), (13, 0)])
def test_ippd_masked_prompt_equals_standard_prompting(seed, lp):
    """Sec. 4.2: attn_IPPD == attn_AR.  Literal stacked prompt with dense mask, pads for
    stopped questions and a shared instruction vs independent standard prompting."""
    c = _small_case(seed, lp=lp)
    nt = len(c["seg_len"])
    act = rng(seed + 100).random(nt) < 0.7
    act[0] = True
    qlen = np.minimum(c["seg_len"], rng(seed + 200).integers(1, 3, size=nt))
    st = O.KVState(list(c["sk"]), list(c["sv"]))
    o2, l2 = O.stacked_prompt_step(c["ck"], c["cv"], c["ctx_start"], c["q_start"], st, qlen,
                                   c["q"], c["k"], c["v"], act, 10000.0,
                                   instr_k=c["ik"], instr_v=c["iv"])
    prompt_of = np.searchsorted(c["q_start"], np.arange(nt), side="right") - 1
    for i in range(nt):
        if not act[i]:
            assert np.isnan(o2[i]).all()
            continue
        b = prompt_of[i]
        sl = slice(c["ctx_start"][b], c["ctx_start"][b + 1])
        o1, l1 = O.standard_prompting_question(c["ck"][sl], c["cv"][sl], c["sk"][i], c["sv"][i],
                                               c["q"][i], c["k"][i], c["v"][i], 10000.0,
                                               instr_k=c["ik"], instr_v=c["iv"])
        np.testing.assert_allclose(o2[i], o1, atol=1e-12)
        np.testing.assert_allclose(l2[i], l1, atol=1e-12)


def test_two_level_batch_matches_stacked_prompts():
    """Two-level batch (Sec. 4.4): prompts 0-1 behind instruction 0 and prompt 2
    behind instruction 1.  The per-question oracle with per-prompt
    instructions equals, for each instruction, the literal stacked prompt of
    that instruction and its contexts under the dense mask."""
    c = _small_case(31, B=3)
    r = rng(32)
    hkv, d = 2, 16
    lps = [4, 3]
    ik = [r.standard_normal((n, hkv, d)) for n in lps]
    iv = [r.standard_normal((n, hkv, d)) for n in lps]
    instr = O.Instructions(np.array([0, 2, 3]), np.array([0, 4, 7]), np.concatenate(ik), np.concatenate(iv))
    nt = len(c["seg_len"])
    act = np.ones(nt, bool)
    act[-1] = False
    out, lse = O.decode_step_standard(c["ck"], c["cv"], c["ctx_start"], c["q_start"],
                                      O.KVState(list(c["sk"]), list(c["sv"])), c["q"], c["k"], c["v"], act,
                                      1e4, instr=instr)
    for s, (b0, b1) in enumerate([(0, 2), (2, 3)]):
        q0, q1 = c["q_start"][b0], c["q_start"][b1]
        cs = c["ctx_start"][b0:b1 + 1] - c["ctx_start"][b0]
        qs = c["q_start"][b0:b1 + 1] - q0
        ctx = slice(c["ctx_start"][b0], c["ctx_start"][b1])
        st = O.KVState(list(c["sk"][q0:q1]), list(c["sv"][q0:q1]))
        o2, l2 = O.stacked_prompt_step(c["ck"][ctx], c["cv"][ctx], cs, qs, st, c["seg_len"][q0:q1],
                                       c["q"][q0:q1], c["k"][q0:q1], c["v"][q0:q1], act[q0:q1], 1e4,
                                       instr_k=ik[s], instr_v=iv[s])
        np.testing.assert_allclose(np.nan_to_num(out[q0:q1]), np.nan_to_num(o2), atol=1e-12)
        np.testing.assert_allclose(np.nan_to_num(lse[q0:q1]), np.nan_to_num(l2), atol=1e-12)
    assert np.isnan(out[-1]).all()


def test_batched_step_matches_per_question():
    c = _small_case(20, B=3)
    nt = len(c["seg_len"])
    act = np.ones(nt, bool); act[1] = False
    st = O.KVState(list(c["sk"]), list(c["sv"]))
    out, lse = O.decode_step_standard(c["ck"], c["cv"], c["ctx_start"], c["q_start"], st,
                                      c["q"], c["k"], c["v"], act, 1e4)
    assert np.isnan(out[1]).all() and np.isnan(lse[1]).all()
    qlen = c["seg_len"]
    o2, _ = O.stacked_prompt_step(c["ck"], c["cv"], c["ctx_start"], c["q_start"],
                                  O.KVState(list(c["sk"]), list(c["sv"])), qlen,
                                  c["q"], c["k"], c["v"], act, 1e4)
    np.testing.assert_allclose(np.nan_to_num(out), np.nan_to_num(o2), atol=1e-12)


def test_question_permutation_equivariance():
    """Answers are independent (Sec. 3): permuting a prompt's questions permutes outputs."""
    c = _small_case(30, B=1, nq=(4, 4))
    nt = len(c["seg_len"])
    act = np.ones(nt, bool)
    perm = np.array([2, 0, 3, 1])
    st = O.KVState(list(c["sk"]), list(c["sv"]))
    out, _ = O.decode_step_standard(c["ck"], c["cv"], c["ctx_start"], c["q_start"], st,
                                    c["q"], c["k"], c["v"], act, 1e4)
    st2 = O.KVState([c["sk"][p] for p in perm], [c["sv"][p] for p in perm])
    out2, _ = O.decode_step_standard(c["ck"], c["cv"], c["ctx_start"], c["q_start"], st2,
                                     c["q"][perm], c["k"][perm], c["v"][perm], act, 1e4)
    np.testing.assert_array_equal(out2, out[perm])


def test_no_cross_question_or_cross_context_leakage():
    """Sec. 4.1: an answer token sees only p, its context, its question and its own answer."""
    c = _small_case(40, B=2, nq=(2, 2))
    act = np.ones(4, bool)
    qlen = np.ones(4, int)
    base = O.stacked_prompt_step(c["ck"], c["cv"], c["ctx_start"], c["q_start"],
                                 O.KVState(list(c["sk"]), list(c["sv"])), qlen,
                                 c["q"], c["k"], c["v"], act, 1e4)[0]
    # perturb question 1's segment and new token, and prompt 1's context
    sk = list(c["sk"]); sk[1] = sk[1] + 5.0
    k = c["k"].copy(); k[1] += 3.0
    ck = c["ck"].copy(); ck[c["ctx_start"][1]:] += 7.0
    pert = O.stacked_prompt_step(ck, c["cv"], c["ctx_start"], c["q_start"],
                                 O.KVState(sk, list(c["sv"])), qlen,
                                 c["q"], k, c["v"], act, 1e4)[0]
    np.testing.assert_array_equal(pert[0], base[0])      # question 0 of prompt 0 unaffected
    assert not np.allclose(pert[1], base[1])
    assert not np.allclose(pert[2], base[2])


def test_mask_fixture_hand_derived():
    meta_lines = {}
    rows = {}
    with open(os.path.join(GOLDEN, "stacked_mask_example.txt")) as f:
        for line in f:
            line = line.strip()
            if not line or line.startswith("#"):
                continue
            key, *vals = line.split()
            if key == "row":
                rows[int(vals[0])] = np.array(vals[1:], dtype=int).astype(bool)
            else:
                meta_lines[key] = [int(v) for v in vals]
    meta = O.build_stacked_metadata(meta_lines["lp"][0], meta_lines["ctx_len"],
                                    meta_lines["q_start"], meta_lines["question_len"],
                                    meta_lines["fed_len"],
                                    [bool(a) for a in meta_lines["active"]])
    np.testing.assert_array_equal(meta.pos, meta_lines["pos"])
    np.testing.assert_array_equal(meta.ctx, meta_lines["ctx"])
    np.testing.assert_array_equal(meta.qtn, meta_lines["qtn"])
    got = O.mask_predicates(meta, np.array(sorted(rows)))
    for r_i, r in enumerate(sorted(rows)):
        np.testing.assert_array_equal(got[r_i], rows[r])


# ----------------------------------------------------------- brute force ---

def brute_force_mp(ctx_k, ctx_v, seg_k, seg_v, qn, kn, vn, base, dps=50):
    """50-digit evaluation: rotation as complex exponential, softmax by definition."""
    mpmath.mp.dps = dps
    K = [list(map(lambda r: [mpmath.mpf(float(x)) for x in r], t))
         for t in np.concatenate([ctx_k, seg_k, kn[None]])]
    V = np.concatenate([ctx_v, seg_v, vn[None]])
    n, hkv, d = len(K), ctx_k.shape[1], ctx_k.shape[2]
    hq = qn.shape[0]
    h2 = d // 2

    def rot(vec, m):
        res = [None] * d
        for j in range(h2):
            th = mpmath.power(mpmath.mpf(base), -mpmath.mpf(2 * j) / d)
            z = mpmath.mpc(vec[j], vec[j + h2]) * mpmath.expj(m * th)
            res[j], res[j + h2] = z.real, z.imag
        return res

    out = np.zeros((hq, d))
    for h in range(hq):
        g = h * hkv // hq
        q = rot([mpmath.mpf(float(x)) for x in qn[h]], n - 1)
        logits = []
        for t in range(n):
            kr = rot(K[t][g], t)
            logits.append(mpmath.fsum(a * b for a, b in zip(q, kr)) / mpmath.sqrt(d))
        mx = max(logits)
        w = [mpmath.exp(x - mx) for x in logits]
        tot = mpmath.fsum(w)
        for j in range(d):
            out[h, j] = float(mpmath.fsum(w[t] * mpmath.mpf(float(V[t, g, j])) for t in range(n)) / tot)
    return out


@pytest.mark.parametrize("lc,s,d", [(1, 0, 2), (2, 1, 4), (3, 2, 4)])
def test_brute_force_tiny(lc, s, d):
    r = rng(50 + lc)
    hq, hkv = 2, 1
    ck, cv = r.standard_normal((2, lc, hkv, d))
    sk, sv = r.standard_normal((2, s, hkv, d))
    qn = r.standard_normal((hq, d))
    kn, vn = r.standard_normal((2, hkv, d))
    out, _ = O.standard_prompting_question(ck, cv, sk, sv, qn, kn, vn, 10.0)
    ref = brute_force_mp(ck, cv, sk, sv, qn, kn, vn, 10.0)
    np.testing.assert_allclose(out, ref, atol=1e-14)


# ------------------------------------------------------------ multi-step ---

def test_decode_run_segments_follow_stop_steps():
    """Sec. 4.2: stopped answers receive no further tokens; active ones grow by one per step."""
    wl = W.custom_workload(num_prompts=2, questions=(3, 3), seg_len=(2, 5), steps=4,
                           stop=(1, 4), ctx_len=(6, 9))
    st = W.make_structure(wl)
    kv = W.layer_kv(st)
    state = O.KVState.from_packed(kv.seg_k, kv.seg_v, st.seg_start)
    steps = [W.step_inputs(st, t) for t in range(wl.steps)]
    res = O.decode_run(kv.ctx_k, kv.ctx_v, st.ctx_start, st.q_start, state,
                       [(s.q_new, s.k_new, s.v_new, s.active) for s in steps], wl.rope_base)
    np.testing.assert_array_equal(state.seg_len(), st.seg_len_at(wl.steps))
    for t in range(wl.steps):
        out, _ = res[t]
        np.testing.assert_array_equal(np.isnan(out[:, 0, 0]), ~st.active(t))


def test_decode_run_step_token_is_last_key():
    """After a step the fed token sits in its segment: step t+1 equals a single step from
    a state whose segment already holds it (positions continue, Sec. 4.1)."""
    wl = W.custom_workload(questions=(2, 2), seg_len=(3, 3), steps=2)
    st = W.make_structure(wl)
    kv = W.layer_kv(st)
    s0, s1 = W.step_inputs(st, 0), W.step_inputs(st, 1)
    state = O.KVState.from_packed(kv.seg_k, kv.seg_v, st.seg_start)
    res = O.decode_run(kv.ctx_k, kv.ctx_v, st.ctx_start, st.q_start, state,
                       [(s.q_new, s.k_new, s.v_new, s.active) for s in (s0, s1)], wl.rope_base)
    seg_k = [np.concatenate([kv.seg_k[st.seg_start[i]:st.seg_start[i + 1]], s0.k_new[i][None]])
             for i in range(2)]
    seg_v = [np.concatenate([kv.seg_v[st.seg_start[i]:st.seg_start[i + 1]], s0.v_new[i][None]])
             for i in range(2)]
    for i in range(2):
        o, _ = O.standard_prompting_question(kv.ctx_k, kv.ctx_v, seg_k[i], seg_v[i],
                                             s1.q_new[i], s1.k_new[i], s1.v_new[i], wl.rope_base)
        np.testing.assert_array_equal(res[1][0][i], o)


# ------------------------------------------------------ planted mistakes ---

def _sdpa_pin_passes():
    try:
        test_single_question_is_causal_attention_sdpa()
        return True
    except AssertionError:
        return False


def _masked_pin_passes():
    try:
        test_ippd_masked_prompt_equals_standard_prompting(11, 3)
        return True
    except AssertionError:
        return False


def test_planted_mistakes_are_caught(monkeypatch):
    """Plausible oracle slips each fail at least one pin (the mistake is planted in the
    oracle, on the CPU)."""
    good_rope, good_attend = O.rope, O.attend

    # 1. rotation sign flipped
    monkeypatch.setattr(O, "rope", lambda x, p, b: good_rope(x, -np.asarray(p), b))
    assert not _sdpa_pin_passes()
    monkeypatch.setattr(O, "rope", good_rope)

    # 2. decode query one position too early (off-by-one in the virtual position)
    orig_spq = O.standard_prompting_question

    def early(ctx_k, ctx_v, seg_k, seg_v, q_new, k_new, v_new, base, scale=None, **kw):
        qs = good_rope(np.asarray(q_new, float), -1, base)   # net position n-2
        return orig_spq(ctx_k, ctx_v, seg_k, seg_v, qs, k_new, v_new, base, scale, **kw)
    monkeypatch.setattr(O, "standard_prompting_question", early)
    assert not _sdpa_pin_passes()
    monkeypatch.setattr(O, "standard_prompting_question", orig_spq)

    # 3. the step's own key dropped from the softmax support
    def drop_last(q, K, V, scale, mask=None):
        if mask is None:
            return good_attend(q, K[:-1], V[:-1], scale)
        return good_attend(q, K, V, scale, mask)
    monkeypatch.setattr(O, "attend", drop_last)
    assert not _sdpa_pin_passes()
    assert not _masked_pin_passes()
    monkeypatch.setattr(O, "attend", good_attend)

    # 4. wrong GQA mapping (h % Hkv instead of h // G): route through an altered oracle
    def bad_gqa(ctx_k, ctx_v, seg_k, seg_v, q_new, k_new, v_new, base, scale=None, **kw):
        hq = q_new.shape[0]
        hkv = k_new.shape[0]
        perm = np.array([(h % hkv) * (hq // hkv) + h // hkv for h in range(hq)])
        o, l = orig_spq(ctx_k, ctx_v, seg_k, seg_v, q_new[perm], k_new, v_new, base, scale, **kw)
        inv = np.argsort(perm)
        return o[inv], l[inv]
    monkeypatch.setattr(O, "standard_prompting_question", bad_gqa)
    assert not _sdpa_pin_passes()
    monkeypatch.setattr(O, "standard_prompting_question", orig_spq)

    # 5. causal predicate written with '>' instead of '>=' (a token not seeing itself)
    good_mp = O.mask_predicates

    def strict(meta, rows):
        m = good_mp(meta, rows)
        m[np.arange(len(rows)), rows] = False
        return m
    monkeypatch.setattr(O, "mask_predicates", strict)
    assert not _masked_pin_passes()
    monkeypatch.setattr(O, "mask_predicates", good_mp)
    assert _sdpa_pin_passes() and _masked_pin_passes()
