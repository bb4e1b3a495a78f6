"""Plain fp64 reference of the stacked-prompt prefill attention (test
infrastructure only: tests, the smoke check and the bench's CPU baseline use
it; the GPU path never does).

The prefill is the forward pass over the prompt header before any answer
token exists (Sec. 4.1).  Every header token is a query row:

* Path 1, *standard prompting* (Sec. 3): each question is its own prompt
  [context; question] at real positions 0..n-1 and every row takes causal
  attention over the keys at or before it.  The context rows do not depend on
  the question (causality), so they are computed once per prompt, from its
  first question's sequence (or the context alone when it has none).

* Path 2, *the literal IPPD prompt* (Sec. 4.1): the header
  [c_1, x_11, x_12, ..., c_2, x_21, ...] with (pos_virt, ctx, qtn) per token,
  the dense mask M_fin = M_caus AND M_ctx AND M_qtn, and one pad per question
  at pos_virt = max int standing in for the answer slots that are still
  empty (Sec. 4.4); each header row takes a softmax over ALL keys with the
  additive 0/-inf mask.

The two are equal (the argument of Sec. 4.2 applies to every row, not only
to decode rows).  Rotary embedding and softmax scale follow the decode
oracle (rotate-half, theta_j = base^(-2j/D), scale 1/sqrt(D)).

Parity pins: tests/test_prefill_oracle.py (torch SDPA in fp64, the decode
oracle at the last question token, prefix closure of causal rows, planted
mistakes).
"""
from __future__ import annotations

from typing import Optional, Sequence

import numpy as np

from . import ippd as O


def standard_prefill_question(ctx_k, ctx_v, ctx_q, seg_k, seg_v, seg_q, base: float,
                              scale: Optional[float] = None, rows: Optional[Sequence[int]] = None,
                              instr=None):
    """Path 1 for one question: causal attention over [instruction; context; question].

    ctx_* are raw [Lc, H, D] (keys/values with Hkv heads, queries with Hq);
    seg_* the question's raw tokens [s, H, D]; ``instr`` optionally
    (k, v, q) of an instruction p placed before the context (Sec. 4.1: p at
    [0, |p|)).  ``rows`` selects sequence positions to compute (default all
    n = |p| + Lc + s).  Returns out [n, Hq, D] (NaN for rows not computed).
    """
    parts = ([instr] if instr is not None else []) + [(ctx_k, ctx_v, ctx_q), (seg_k, seg_v, seg_q)]
    K = np.concatenate([np.asarray(x[0], np.float64) for x in parts], axis=0)
    V = np.concatenate([np.asarray(x[1], np.float64) for x in parts], axis=0)
    Q = np.concatenate([np.asarray(x[2], np.float64) for x in parts], axis=0)
    n, hkv, d = K.shape
    hq = Q.shape[1]
    G = hq // hkv
    if scale is None:
        scale = 1.0 / np.sqrt(d)
    pos = np.arange(n)
    Kr = O.rope(K.transpose(1, 0, 2), pos, base)            # [Hkv, n, D]
    out = np.full((n, hq, d), np.nan)
    for t in (range(n) if rows is None else rows):
        qr = O.rope(Q[t], t, base)                          # [Hq, D] at real position t
        for h in range(hq):
            g = h // G
            out[t, h], _ = O.attend(qr[h], Kr[g, : t + 1], V[: t + 1, g], scale)
    return out


def prefill_standard(ctx_k, ctx_v, ctx_q, ctx_start, q_start, seg_k, seg_v, seg_q, seg_start,
                     base: float, scale: Optional[float] = None, ctx_rows=None, seg_rows=None,
                     instr=None):
    """Path 1 over a ragged batch of prompts.

    Packed inputs as in the decode oracle: prompt b's context tokens at
    ctx_start[b]:ctx_start[b+1], question i's tokens at seg_start[i]:seg_start[i+1].
    ``instr`` (two-level batch) is (prompt_start, tok_start, k, v, q): prompts
    prompt_start[s]:prompt_start[s+1] sit behind instruction s, whose raw
    tokens are k/v/q[tok_start[s]:tok_start[s+1]]; every question's own
    prompt is then [p_s; c_b; x_i].
    ``ctx_rows`` / ``seg_rows`` optionally list packed token indices to compute.
    Returns out_ctx [sum Lc, Hq, D] and out_seg [sum s, Hq, D] (NaN where not
    computed), and with ``instr`` also out_instr [sum |p|, Hq, D].
    """
    hq, d = ctx_q.shape[1], ctx_q.shape[2]
    B = len(ctx_start) - 1
    out_ctx = np.full((int(ctx_start[-1]), hq, d), np.nan)
    out_seg = np.full((int(seg_start[-1]), hq, d), np.nan)
    want_c = None if ctx_rows is None else set(int(x) for x in ctx_rows)
    want_s = None if seg_rows is None else set(int(x) for x in seg_rows)
    ins_of = (lambda b: None)
    out_ins = None
    if instr is not None:
        pstart, tstart, ik, iv, iq = instr
        out_ins = np.full((int(tstart[-1]), hq, d), np.nan)

        def ins_of(b):
            s_ = int(np.searchsorted(pstart, b, side="right") - 1)
            t0, t1 = int(tstart[s_]), int(tstart[s_ + 1])
            return s_, (ik[t0:t1], iv[t0:t1], iq[t0:t1])
        # instruction rows: causal over the instruction alone
        for s_ in range(len(tstart) - 1):
            t0, t1 = int(tstart[s_]), int(tstart[s_ + 1])
            if t1 > t0:
                e = ik[t0:t0]
                o = standard_prefill_question(ik[t0:t1], iv[t0:t1], iq[t0:t1], e, e, iq[t0:t0], base, scale)
                out_ins[t0:t1] = o
    for b in range(B):
        c0, c1 = int(ctx_start[b]), int(ctx_start[b + 1])
        lc = c1 - c0
        ins = ins_of(b)
        pre = None if ins is None else ins[1]
        lp = 0 if pre is None else len(pre[0])
        qs = range(int(q_start[b]), int(q_start[b + 1]))
        # context rows: causal over [instruction; context] (the same in every question's prompt)
        rows = [lp + t for t in range(lc) if want_c is None or c0 + t in want_c]
        if rows:
            o = standard_prefill_question(ctx_k[c0:c1], ctx_v[c0:c1], ctx_q[c0:c1],
                                          ctx_k[c0:c0], ctx_v[c0:c0], ctx_q[c0:c0], base, scale, rows, pre)
            out_ctx[c0 + np.asarray(rows) - lp] = o[rows]
        for i in qs:
            s0, s1 = int(seg_start[i]), int(seg_start[i + 1])
            rows = [lp + lc + u for u in range(s1 - s0) if want_s is None or s0 + u in want_s]
            if not rows:
                continue
            o = standard_prefill_question(ctx_k[c0:c1], ctx_v[c0:c1], ctx_q[c0:c1],
                                          seg_k[s0:s1], seg_v[s0:s1], seg_q[s0:s1], base, scale, rows, pre)
            out_seg[s0 + np.asarray(rows) - lp - lc] = o[rows]
    if instr is not None:
        return out_ctx, out_seg, out_ins
    return out_ctx, out_seg


def stacked_prefill(ctx_k, ctx_v, ctx_q, ctx_start, q_start, seg_k, seg_v, seg_q, seg_start,
                    base: float, scale: Optional[float] = None, instr=None):
    """Path 2: every header row of the literal stacked prompt under M_fin.

    ``instr`` optionally (k, v, q) of one instruction p shared by all the
    contexts of this stacked prompt (ctx = 0 tokens at [0, |p|), Sec. 4.1).
    Returns out_ctx [sum Lc, Hq, D] and out_seg [sum s, Hq, D] (and out_instr
    [|p|, Hq, D] with ``instr``).
    """
    hkv, d = ctx_k.shape[1], ctx_k.shape[2]
    hq = ctx_q.shape[1]
    G = hq // hkv
    if scale is None:
        scale = 1.0 / np.sqrt(d)
    B = len(ctx_start) - 1
    nt = int(q_start[-1])
    ctx_len = [int(ctx_start[b + 1] - ctx_start[b]) for b in range(B)]
    qlen = [int(seg_start[i + 1] - seg_start[i]) for i in range(nt)]
    # no answer token exists yet: every question's slot in the step round is a pad
    lp = 0 if instr is None else len(instr[0])
    meta = O.build_stacked_metadata(lp, ctx_len, list(q_start), qlen, [0] * nt, [False] * nt)
    n = len(meta.src)
    K = np.zeros((n, hkv, d))
    V = np.zeros((n, hkv, d))
    Q = np.zeros((n, hq, d))
    header = []
    for t, (kind, owner, idx) in enumerate(meta.src):
        if kind == "instr":
            K[t], V[t], Q[t] = instr[0][idx], instr[1][idx], instr[2][idx]
            header.append((t, "instr", idx))
        elif kind == "ctx":
            j = int(ctx_start[owner]) + idx
            K[t], V[t], Q[t] = ctx_k[j], ctx_v[j], ctx_q[j]
            header.append((t, "ctx", j))
        elif kind == "seg":
            j = int(seg_start[owner]) + idx
            K[t], V[t], Q[t] = seg_k[j], seg_v[j], seg_q[j]
            header.append((t, "seg", j))
        # pads keep zero keys and values: M_caus never lets a header row see them
    Kr = O.rope(K.transpose(1, 0, 2), meta.pos.astype(np.float64)[None, :], base)
    rows = np.array([t for t, _, _ in header], dtype=np.int64)
    add_mask = np.where(O.mask_predicates(meta, rows), 0.0, -np.inf)
    out_ctx = np.full((int(ctx_start[-1]), hq, d), np.nan)
    out_seg = np.full((int(seg_start[-1]), hq, d), np.nan)
    out_ins = np.full((lp, hq, d), np.nan)
    for r, (t, kind, j) in enumerate(header):
        qr = O.rope(Q[t], meta.pos[t], base)
        dst = {"ctx": out_ctx, "seg": out_seg, "instr": out_ins}[kind]
        for h in range(hq):
            dst[j, h], _ = O.attend(qr[h], Kr[h // G], V[:, h // G, :], scale, add_mask[r])
    if instr is not None:
        return out_ctx, out_seg, out_ins
    return out_ctx, out_seg
