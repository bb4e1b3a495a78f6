"""Pins of the prefill oracle against what the paper and mathematics fix.

None compares the oracle with itself: torch SDPA in fp64 (a library routine)
for the causal rows, the decode oracle (pinned in test_oracle_pins.py) at the
last question token, the literal stacked prompt under M_fin, and the prefix
closure of causal attention.  The planted-mistake test shows that plausible
slips fail a pin.
"""
import numpy as np
import pytest
import torch

from oracle import ippd as O
from oracle import prefill as P
import workload as W

from tests.test_oracle_pins import rope_complex


def _case(seed, ctx_lens, q_counts, hq=8, hkv=2, d=32, qlen=(2, 6)):
    r = np.random.default_rng(seed)
    ctx_start = np.concatenate([[0], np.cumsum(ctx_lens)]).astype(int)
    q_start = np.concatenate([[0], np.cumsum(q_counts)]).astype(int)
    nt = int(q_start[-1])
    sl = r.integers(qlen[0], qlen[1], size=nt, endpoint=True)
    seg_start = np.concatenate([[0], np.cumsum(sl)]).astype(int)
    nc, ns = int(ctx_start[-1]), int(seg_start[-1])
    return dict(ck=r.standard_normal((nc, hkv, d)), cv=r.standard_normal((nc, hkv, d)),
                cq=r.standard_normal((nc, hq, d)), sk=r.standard_normal((ns, hkv, d)),
                sv=r.standard_normal((ns, hkv, d)), sq=r.standard_normal((ns, hq, d)),
                ctx_start=ctx_start, q_start=q_start, seg_start=seg_start)


def _standard(c, base=10000.0):
    return P.prefill_standard(c["ck"], c["cv"], c["cq"], c["ctx_start"], c["q_start"], c["sk"], c["sv"],
                              c["sq"], c["seg_start"], base)


def test_prefill_rows_are_causal_attention_sdpa():
    """Every row of one question's prompt [context; question] is a row of causal
    attention at real positions: torch SDPA (fp64, GQA, is_causal) on keys and
    queries rotated by the complex form of the rotary map."""
    c = _case(1, [11], [1], qlen=(6, 6))
    base = 10000.0
    oc, os_ = _standard(c, base)
    K = np.concatenate([c["ck"], c["sk"]])
    V = np.concatenate([c["cv"], c["sv"]])
    Q = np.concatenate([c["cq"], c["sq"]])
    n = len(K)
    Kr = np.stack([rope_complex(K[t], t, base) for t in range(n)])
    Qr = np.stack([rope_complex(Q[t], t, base) for t in range(n)])
    qt, kt, vt = (torch.from_numpy(a).permute(1, 0, 2)[None] for a in (Qr, Kr, V))
    ref = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, is_causal=True, enable_gqa=True)
    ref = ref[0].permute(1, 0, 2).numpy()                      # [n, Hq, D]
    np.testing.assert_allclose(np.concatenate([oc, os_]), ref, atol=1e-12)


def test_last_question_token_is_a_decode_step():
    """The prefill row of a question's last token equals the decode oracle with
    that token as the step's token over the earlier ones as the cached segment."""
    c = _case(2, [9, 14], [2, 3])
    _, os_ = _standard(c)
    for i in range(int(c["q_start"][-1])):
        b = int(np.searchsorted(c["q_start"], i, side="right") - 1)
        c0, c1 = c["ctx_start"][b], c["ctx_start"][b + 1]
        s0, s1 = c["seg_start"][i], c["seg_start"][i + 1]
        out, _ = O.standard_prompting_question(c["ck"][c0:c1], c["cv"][c0:c1], c["sk"][s0:s1 - 1],
                                               c["sv"][s0:s1 - 1], c["sq"][s1 - 1], c["sk"][s1 - 1],
                                               c["sv"][s1 - 1], 10000.0)
        np.testing.assert_allclose(os_[s1 - 1], out, atol=1e-12)


@pytest.mark.parametrize("seed", [3, 4])
def test_stacked_prompt_equals_standard_prompting(seed):
    """Sec. 4.2 for every header row: the literal stacked prompt under M_fin
    (pads at max int) equals per-question standard prompting."""
    c = _case(seed, [7, 12, 5], [3, 1, 2])
    a = _standard(c)
    b = P.stacked_prefill(c["ck"], c["cv"], c["cq"], c["ctx_start"], c["q_start"], c["sk"], c["sv"], c["sq"],
                          c["seg_start"], 10000.0)
    np.testing.assert_allclose(a[0], b[0], atol=1e-12)
    np.testing.assert_allclose(a[1], b[1], atol=1e-12)


@pytest.mark.parametrize("seed", [7, 8])
def test_two_level_prefill_equals_stacked_prompt(seed):
    """Two-level prefill (Sec. 4.4): one instruction shared by every context of the
    stacked prompt.  Per-question standard prompting [p; c_b; x_i] equals the
    literal stacked header under M_fin, instruction rows included."""
    c = _case(seed, [6, 9, 4], [2, 1, 3])
    r = np.random.default_rng(seed + 50)
    lp = 5
    ik, iv = r.standard_normal((2, lp, 2, 32))
    iq = r.standard_normal((lp, 8, 32))
    a = P.prefill_standard(c["ck"], c["cv"], c["cq"], c["ctx_start"], c["q_start"], c["sk"], c["sv"], c["sq"],
                           c["seg_start"], 10000.0, instr=(np.array([0, 3]), np.array([0, lp]), ik, iv, iq))
    b = P.stacked_prefill(c["ck"], c["cv"], c["cq"], c["ctx_start"], c["q_start"], c["sk"], c["sv"], c["sq"],
                          c["seg_start"], 10000.0, instr=(ik, iv, iq))
    for x, y in zip(a, b):
        np.testing.assert_allclose(x, y, atol=1e-12)


def test_two_level_prefill_rows_are_causal_attention_sdpa():
    """One question's prompt [p; c; x]: every row is causal attention at real
    positions (torch SDPA in fp64, keys and queries rotated by the complex form)."""
    c = _case(9, [7], [1], qlen=(4, 4))
    r = np.random.default_rng(60)
    lp = 6
    ik, iv = r.standard_normal((2, lp, 2, 32))
    iq = r.standard_normal((lp, 8, 32))
    oc, os_, oi = P.prefill_standard(c["ck"], c["cv"], c["cq"], c["ctx_start"], c["q_start"], c["sk"], c["sv"],
                                     c["sq"], c["seg_start"], 10000.0,
                                     instr=(np.array([0, 1]), np.array([0, lp]), ik, iv, iq))
    K = np.concatenate([ik, c["ck"], c["sk"]])
    V = np.concatenate([iv, c["cv"], c["sv"]])
    Q = np.concatenate([iq, c["cq"], c["sq"]])
    n = len(K)
    Kr = np.stack([rope_complex(K[t], t, 10000.0) for t in range(n)])
    Qr = np.stack([rope_complex(Q[t], t, 10000.0) for t in range(n)])
    qt, kt, vt = (torch.from_numpy(a).permute(1, 0, 2)[None] for a in (Qr, Kr, V))
    ref = torch.nn.functional.scaled_dot_product_attention(qt, kt, vt, is_causal=True, enable_gqa=True)
    ref = ref[0].permute(1, 0, 2).numpy()
    np.testing.assert_allclose(np.concatenate([oi, oc, os_]), ref, atol=1e-12)


def test_context_rows_ignore_the_questions_and_rows_are_prefix_closed():
    """Causality: a context row does not change when questions (or later context
    tokens) are appended; it equals the same row of a prefill of the prefix alone."""
    c = _case(5, [10], [2])
    oc, _ = _standard(c)
    pre = P.standard_prefill_question(c["ck"][:6], c["cv"][:6], c["cq"][:6], c["ck"][:0], c["cv"][:0],
                                      c["cq"][:0], 10000.0)
    np.testing.assert_allclose(oc[:6], pre, atol=1e-15)


def test_row_selection_matches_full():
    c = _case(6, [8, 6], [2, 2])
    full = _standard(c)
    part = P.prefill_standard(c["ck"], c["cv"], c["cq"], c["ctx_start"], c["q_start"], c["sk"], c["sv"],
                              c["sq"], c["seg_start"], 10000.0, ctx_rows=[0, 7, 13], seg_rows=[1, 5])
    np.testing.assert_array_equal(part[0][[0, 7, 13]], full[0][[0, 7, 13]])
    np.testing.assert_array_equal(part[1][[1, 5]], full[1][[1, 5]])
    assert np.isnan(part[0][1]).all() and np.isnan(part[1][0]).all()


def test_prefill_queries_stream_is_seeded_and_separate():
    wl = W.custom_workload(wid=71, dtype="bf16", ctx_len=(9, 9), questions=(2, 2), question_tokens=3,
                           seg_len=(0, 0))
    st = W.make_structure(wl)
    a, b = W.prefill_queries(st), W.prefill_queries(st)
    np.testing.assert_array_equal(a.ctx_q, b.ctx_q)
    assert a.ctx_q.shape == (9, wl.hq, wl.head_dim) and a.seg_q.shape == (6, wl.hq, wl.head_dim)
    assert np.array_equal(W.round_to_bf16(a.seg_q), a.seg_q)
    kv = W.layer_kv(st)
    assert not np.array_equal(a.ctx_q[:, : wl.hkv], kv.ctx_k)


# ------------------------------------------------------ planted mistakes ---

def _passes(fn, *a):
    try:
        fn(*a)
        return True
    except AssertionError:
        return False


def test_planted_mistakes_are_caught(monkeypatch):
    good_spq = P.standard_prefill_question

    # 1. causal window one key short (a row not seeing itself)
    def short(ctx_k, ctx_v, ctx_q, seg_k, seg_v, seg_q, base, scale=None, rows=None, instr=None):
        out = good_spq(ctx_k, ctx_v, ctx_q, seg_k, seg_v, seg_q, base, scale, rows, instr)
        n = len(ctx_k) + len(seg_k) + (0 if instr is None else len(instr[0]))
        for t in (range(n) if rows is None else rows):
            if t > 0:
                o = good_spq(ctx_k, ctx_v, ctx_q, seg_k, seg_v, seg_q, base, scale, [t - 1], instr)
                out[t] = o[t - 1]
        return out
    monkeypatch.setattr(P, "standard_prefill_question", short)
    assert not _passes(test_prefill_rows_are_causal_attention_sdpa)
    assert not _passes(test_two_level_prefill_rows_are_causal_attention_sdpa)
    monkeypatch.setattr(P, "standard_prefill_question", good_spq)

    # 1b. the instruction dropped from the context and question rows' prompts
    def no_instr(ctx_k, ctx_v, ctx_q, seg_k, seg_v, seg_q, base, scale=None, rows=None, instr=None):
        lp = 0 if instr is None else len(instr[0])
        o = good_spq(ctx_k, ctx_v, ctx_q, seg_k, seg_v, seg_q, base, scale,
                     None if rows is None else [t - lp for t in rows])
        return np.concatenate([np.full((lp,) + o.shape[1:], np.nan), o])
    monkeypatch.setattr(P, "standard_prefill_question", no_instr)
    assert not _passes(test_two_level_prefill_rows_are_causal_attention_sdpa)
    monkeypatch.setattr(P, "standard_prefill_question", good_spq)

    # 2. question tokens placed one position late (positions Lc+1 ..)
    good_rope = O.rope

    def shifted(x, pos, base):
        return good_rope(x, np.asarray(pos) + (np.asarray(pos) >= 11), base)
    monkeypatch.setattr(O, "rope", shifted)
    assert not _passes(test_prefill_rows_are_causal_attention_sdpa)
    monkeypatch.setattr(O, "rope", good_rope)

    # 3. M_qtn dropped from the stacked mask (questions see each other)
    good_mp = O.mask_predicates

    def no_qtn(meta, rows):
        pq, pk = meta.pos[rows][:, None], meta.pos[None, :]
        cq, ck = meta.ctx[rows][:, None], meta.ctx[None, :]
        return (pq >= pk) & ((cq == ck) | (ck == 0))
    monkeypatch.setattr(O, "mask_predicates", no_qtn)
    assert not _passes(test_stacked_prompt_equals_standard_prompting, 3)
    monkeypatch.setattr(O, "mask_predicates", good_mp)
    assert _passes(test_prefill_rows_are_causal_attention_sdpa)
