"""Plain fp64 reference of one IPPD decode step (test infrastructure only).

Two independent formulations of the same result:

* Path 1, *standard prompting* (Sec. 3, the autoregressive loop
  y_t = f(p, c_j, x_jk, y_<t); Sec. 4.2, attn_AR): every question is decoded
  in isolation as causal attention over the sequence
  [instruction; context; its question+answer segment; the new token] at real
  positions 0..n-1.  Under the causal mask every earlier key is visible, so
  the decode row attends to all n keys, itself included.

* Path 2, *the literal IPPD prompt* (Sec. 4.1): all contexts and questions
  are stacked into one sequence (header then answers appended in step
  order), each token carries (pos_virt, ctx, qtn), the dense mask
  M_fin = M_caus AND M_ctx AND M_qtn is built explicitly, stopped questions
  get a pad token at pos_virt = max int (Sec. 4.4), and each new-token row
  takes a softmax over ALL keys with the additive 0/-inf mask (Sec. 4.2,
  attn_IPPD).

The paper proves attn_IPPD == attn_AR (Sec. 4.2); tests check the two paths
agree to rounding.  Rotary position embedding is the paper's silent
convention (it hands virtual position ids to unchanged models); the reading
used here is the rotate-half form with theta_j = base^(-2j/D), pairs
(j, j + D/2).  Softmax scale is 1/sqrt(d_k) (Sec. 4.2).

Parity pins: see tests/test_oracle_pins.py (closed forms, a library
attention routine, a 50-digit brute force, a hand-derived mask fixture).
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import List, Optional, Sequence, Tuple

import numpy as np

INT_MAX = 2**31 - 1   # pad-token virtual position (Sec. 4.4: "maximum integer value")


# --------------------------------------------------------------------------
# Rotary embedding at a (virtual) position.
# --------------------------------------------------------------------------

def inv_freq(head_dim: int, base: float) -> np.ndarray:
    """theta_j = base^(-2j/D), j = 0..D/2-1, in float64."""
    j = np.arange(head_dim // 2, dtype=np.float64)
    return np.power(np.float64(base), -2.0 * j / head_dim)


def rope(x: np.ndarray, pos, base: float) -> np.ndarray:
    """Rotate-half rotary embedding of x[..., D] at integer positions ``pos``.

    ``pos`` broadcasts against x.shape[:-1].  For pair j: the angle is pos*theta_j and
    (x_j, x_{j+D/2}) -> (x_j cos - x_{j+D/2} sin, x_{j+D/2} cos + x_j sin).
    """
    x = np.asarray(x, dtype=np.float64)
    d = x.shape[-1]
    h = d // 2
    ang = np.asarray(pos, dtype=np.float64)[..., None] * inv_freq(d, base)
    c, s = np.cos(ang), np.sin(ang)
    a, b = x[..., :h], x[..., h:]
    return np.concatenate([a * c - b * s, b * c + a * s], axis=-1)


# --------------------------------------------------------------------------
# One attention row (Sec. 4.2: softmax(q K^T / sqrt(d_k) + M) V).
# --------------------------------------------------------------------------

def attend(q: np.ndarray, K: np.ndarray, V: np.ndarray, scale: float,
           mask: Optional[np.ndarray] = None) -> Tuple[np.ndarray, float]:
    """softmax(scale * K q + M) V for one query; returns (out[D], natural-log lse).

    ``mask`` is the additive mask (0 or -inf) over the keys, or None.
    """
    logits = (K @ q) * scale
    if mask is not None:
        logits = logits + mask
    m = np.max(logits)
    p = np.exp(logits - m)
    l = np.sum(p)
    return (p @ V) / l, float(m + np.log(l))


# --------------------------------------------------------------------------
# Path 1: standard prompting of one question.
# --------------------------------------------------------------------------

def standard_prompting_question(ctx_k, ctx_v, seg_k, seg_v, q_new, k_new, v_new,
                                base: float, scale: Optional[float] = None,
                                instr_k=None, instr_v=None):
    """Decode-row attention of one question run in isolation.

    ctx_* are the raw context keys/values [Lc, Hkv, D]; seg_* the raw
    question+answer segment already in the cache [s, Hkv, D]; q_new [Hq, D],
    k_new/v_new [Hkv, D] belong to the token fed this step.  Optional
    instr_* prepend a shared instruction p.  Positions are the real indices
    of [p; c; seg; new]; the decode query sits at the last one.
    Returns out [Hq, D] and lse [Hq].
    """
    parts_k = [np.asarray(a, np.float64) for a in (instr_k, ctx_k, seg_k) if a is not None]
    parts_v = [np.asarray(a, np.float64) for a in (instr_v, ctx_v, seg_v) if a is not None]
    K = np.concatenate(parts_k + [np.asarray(k_new, np.float64)[None]], axis=0)
    V = np.concatenate(parts_v + [np.asarray(v_new, np.float64)[None]], axis=0)
    n, hkv, d = K.shape
    hq = q_new.shape[0]
    G = hq // hkv
    if scale is None:
        scale = 1.0 / np.sqrt(d)
    pos = np.arange(n)
    Kr = rope(K.transpose(1, 0, 2), pos, base)             # [Hkv, n, D]
    qr = rope(np.asarray(q_new, np.float64), n - 1, base)    # [Hq, D]
    out = np.empty((hq, d))
    lse = np.empty(hq)
    for h in range(hq):
        g = h // G                                            # contiguous GQA groups
        out[h], lse[h] = attend(qr[h], Kr[g], V[:, g, :], scale)
    return out, lse


@dataclass
class KVState:
    """Per-question segments of raw (pre-rotation) K/V, grown by decode steps."""

    seg_k: List[np.ndarray]   # per question [s_i, Hkv, D]
    seg_v: List[np.ndarray]

    @classmethod
    def from_packed(cls, seg_k, seg_v, seg_start):
        ks = [seg_k[seg_start[i]:seg_start[i + 1]] for i in range(len(seg_start) - 1)]
        vs = [seg_v[seg_start[i]:seg_start[i + 1]] for i in range(len(seg_start) - 1)]
        return cls(ks, vs)

    def seg_len(self) -> np.ndarray:
        return np.array([len(k) for k in self.seg_k], dtype=np.int64)

    def append(self, k_new, v_new, active) -> None:
        """Feed this step's token of every active question (Sec. 4.2: stopped answers
        receive no further tokens)."""
        for i in np.flatnonzero(active):
            self.seg_k[i] = np.concatenate([self.seg_k[i], k_new[i][None]], axis=0)
            self.seg_v[i] = np.concatenate([self.seg_v[i], v_new[i][None]], axis=0)


@dataclass
class Instructions:
    """Instruction blocks of a two-level batch (Sec. 4.4: one stacked prompt
    holds several contexts behind one instruction p): prompts
    prompt_start[s]:prompt_start[s+1] sit behind instruction s, whose raw
    keys/values are k/v[tok_start[s]:tok_start[s+1]]."""

    prompt_start: np.ndarray
    tok_start: np.ndarray
    k: np.ndarray
    v: np.ndarray

    def of_prompt(self, b: int):
        s = int(np.searchsorted(self.prompt_start, b, side="right") - 1)
        t0, t1 = int(self.tok_start[s]), int(self.tok_start[s + 1])
        return self.k[t0:t1], self.v[t0:t1]


def decode_step_standard(ctx_k, ctx_v, ctx_start, q_start, state: KVState,
                         q_new, k_new, v_new, active, base: float,
                         scale: Optional[float] = None, questions=None,
                         instr: Optional[Instructions] = None):
    """Path 1 for every active question of a ragged batch of prompts.

    ctx_k/ctx_v are packed [sum Lc, Hkv, D] with prompt b at
    ctx_start[b]:ctx_start[b+1]; questions of prompt b are
    q_start[b]:q_start[b+1].  The state holds segments *before* this step.
    With ``instr``, each question's own prompt is [p_s; c_b; segment] for the
    instruction s that prompt b sits behind.
    Returns out [Nt, Hq, D] and lse [Nt, Hq]; rows of inactive (or
    unrequested) questions are NaN.
    """
    nt = len(state.seg_k)
    hq, d = q_new.shape[1], q_new.shape[2]
    out = np.full((nt, hq, d), np.nan)
    lse = np.full((nt, hq), np.nan)
    which = range(nt) if questions is None else questions
    prompt_of = np.searchsorted(np.asarray(q_start), np.arange(nt), side="right") - 1
    for i in which:
        if not active[i]:
            continue
        b = prompt_of[i]
        c0, c1 = ctx_start[b], ctx_start[b + 1]
        ik, iv = instr.of_prompt(b) if instr is not None else (None, None)
        out[i], lse[i] = standard_prompting_question(
            ctx_k[c0:c1], ctx_v[c0:c1], state.seg_k[i], state.seg_v[i],
            q_new[i], k_new[i], v_new[i], base, scale, instr_k=ik, instr_v=iv)
    return out, lse


# --------------------------------------------------------------------------
# Path 2: the literal stacked prompt with virtual positions and dense mask.
# --------------------------------------------------------------------------

@dataclass
class StackedMeta:
    pos: np.ndarray     # virtual position id per token
    ctx: np.ndarray     # context id: 0 = shared instruction p, j+1 = context c_j
    qtn: np.ndarray     # question id: 0 = p or context token, i+1 = question i
    src: List[Tuple[str, int, int]]   # ("instr"|"ctx"|"seg"|"new"|"pad", owner, index)


def build_stacked_metadata(lp: int, ctx_len: Sequence[int], q_start: Sequence[int],
                           question_len: Sequence[int], fed_len: Sequence[int],
                           active: Sequence[bool]) -> StackedMeta:
    """Token order and (pos_virt, ctx, qtn) of the stacked prompt (Sec. 4.1).

    Header: [p, c_1, x_11, x_12, ..., c_2, x_21, ...].  Answer tokens already
    fed are appended after the header round by round (round r holds the r-th
    answer token of every question that has one); then this step's tokens:
    one per active question, a pad (pos_virt = INT_MAX) per stopped one
    (Sec. 4.4).  Virtual positions: p -> [0, |p|); c_j -> [|p|, |p|+|c_j|);
    x_jk -> [|p|+|c_j|, |p|+|c_j|+|x_jk|); answer token t of (j,k) ->
    |p|+|c_j|+|x_jk|+(t-1).
    """
    pos, ctx, qtn, src = [], [], [], []
    for t in range(lp):
        pos.append(t); ctx.append(0); qtn.append(0); src.append(("instr", 0, t))
    B = len(ctx_len)
    prompt_of = {}
    for b in range(B):
        for t in range(ctx_len[b]):
            pos.append(lp + t); ctx.append(b + 1); qtn.append(0); src.append(("ctx", b, t))
        for i in range(q_start[b], q_start[b + 1]):
            prompt_of[i] = b
            for t in range(question_len[i]):
                pos.append(lp + ctx_len[b] + t); ctx.append(b + 1); qtn.append(i + 1)
                src.append(("seg", i, t))
    nt = q_start[B]
    rounds = max(fed_len) if nt else 0
    for r in range(rounds):
        for i in range(nt):
            if fed_len[i] > r:
                b = prompt_of[i]
                pos.append(lp + ctx_len[b] + question_len[i] + r)
                ctx.append(b + 1); qtn.append(i + 1)
                src.append(("seg", i, question_len[i] + r))
    for i in range(nt):
        b = prompt_of[i]
        if active[i]:
            pos.append(lp + ctx_len[b] + question_len[i] + fed_len[i])
            src.append(("new", i, 0))
        else:
            pos.append(INT_MAX)
            src.append(("pad", i, 0))
        ctx.append(b + 1); qtn.append(i + 1)
    return StackedMeta(np.array(pos, dtype=np.int64), np.array(ctx), np.array(qtn), src)


def mask_predicates(meta: StackedMeta, rows: np.ndarray) -> np.ndarray:
    """Boolean M_fin[q, k] for query tokens ``rows`` against every key (Sec. 4.1).

    M_caus: pos(q) >= pos(k); M_ctx: ctx(q) == ctx(k) or ctx(k) == 0;
    M_qtn: qtn(q) == qtn(k) or qtn(k) == 0.
    """
    pq, cq, qq = meta.pos[rows][:, None], meta.ctx[rows][:, None], meta.qtn[rows][:, None]
    pk, ck, qk = meta.pos[None, :], meta.ctx[None, :], meta.qtn[None, :]
    caus = pq >= pk
    mctx = (cq == ck) | (ck == 0)
    mqtn = (qq == qk) | (qk == 0)
    return caus & mctx & mqtn


def stacked_prompt_step(ctx_k, ctx_v, ctx_start, q_start, state: KVState, question_len,
                        q_new, k_new, v_new, active, base: float,
                        scale: Optional[float] = None, instr_k=None, instr_v=None):
    """Path 2: one decode step of the literal IPPD prompt.

    ``question_len[i]`` is |x_i|: the first question_len[i] tokens of segment
    i are header question tokens, the rest are answer tokens already fed.
    Returns out [Nt, Hq, D], lse [Nt, Hq] (NaN for stopped questions).
    """
    nt = len(state.seg_k)
    hq, d = q_new.shape[1], q_new.shape[2]
    hkv = k_new.shape[1]
    G = hq // hkv
    if scale is None:
        scale = 1.0 / np.sqrt(d)
    B = len(ctx_start) - 1
    ctx_len = [int(ctx_start[b + 1] - ctx_start[b]) for b in range(B)]
    lp = 0 if instr_k is None else len(instr_k)
    seg_len = state.seg_len()
    fed = [int(seg_len[i] - question_len[i]) for i in range(nt)]
    meta = build_stacked_metadata(lp, ctx_len, list(q_start), list(question_len), fed, active)

    n = len(meta.src)
    K = np.empty((n, hkv, d))
    V = np.empty((n, hkv, d))
    new_rows = {}
    for t, (kind, owner, idx) in enumerate(meta.src):
        if kind == "instr":
            K[t], V[t] = instr_k[idx], instr_v[idx]
        elif kind == "ctx":
            K[t], V[t] = ctx_k[ctx_start[owner] + idx], ctx_v[ctx_start[owner] + idx]
        elif kind == "seg":
            K[t], V[t] = state.seg_k[owner][idx], state.seg_v[owner][idx]
        else:   # this step's token, or a pad carrying arbitrary values
            K[t], V[t] = k_new[owner], v_new[owner]
            new_rows[owner] = t
    pos = meta.pos.astype(np.float64)
    Kr = rope(K.transpose(1, 0, 2), pos[None, :], base)      # [Hkv, n, D]

    out = np.full((nt, hq, d), np.nan)
    lse = np.full((nt, hq), np.nan)
    act_ids = [i for i in range(nt) if active[i]]
    rows = np.array([new_rows[i] for i in act_ids], dtype=np.int64)
    if len(rows) == 0:
        return out, lse
    allowed = mask_predicates(meta, rows)
    add_mask = np.where(allowed, 0.0, -np.inf)
    for r, i in enumerate(act_ids):
        qr = rope(np.asarray(q_new[i], np.float64), meta.pos[rows[r]], base)
        for h in range(hq):
            g = h // G
            out[i, h], lse[i, h] = attend(qr[h], Kr[g], V[:, g, :], scale, add_mask[r])
    return out, lse


# --------------------------------------------------------------------------
# Multi-step driver (Sec. 4.2: each step emits one token per active answer,
# which is then appended at its virtual position).
# --------------------------------------------------------------------------

def decode_run(ctx_k, ctx_v, ctx_start, q_start, state: KVState, steps_inputs,
               base: float, scale: Optional[float] = None, record=None,
               instr: Optional[Instructions] = None):
    """Run consecutive decode steps with path 1; returns per-step (out, lse).

    ``steps_inputs`` yields (q_new, k_new, v_new, active) per step.  The
    step's token is attended to (it is the last key) and then stays in its
    segment for later steps.  ``record`` optionally lists the steps to
    return (others are computed only for their appends).
    """
    results = {}
    for t, (q, k, v, act) in enumerate(steps_inputs):
        if record is None or t in record:
            results[t] = decode_step_standard(ctx_k, ctx_v, ctx_start, q_start, state,
                                              q, k, v, act, base, scale, instr=instr)
        state.append(k, v, act)
    return results
