"""Seeded synthetic inputs for the IPPD decode-step attention workloads.

This module is shared by the fp64 oracle and the GPU path.  It holds no
attention or rotary arithmetic: it only draws the raw (pre-rotation) key,
value and query vectors, the ragged lengths and the per-step active flags,
and rounds them to the storage precision so that both sides see identical
numbers.

Workload shapes follow the common-context QA setting of the paper (Sec. 3:
J contexts, M_j questions per context, answers decoded token by token) and
the batch of stacked prompts with different contexts and a shrinking set of
still-decoding questions (Sec. 4.4).  The synthetic recipe, per workload:

* structure stream ``default_rng([wid, 0])``: context length per prompt,
  question count per prompt, initial segment length per question
  (question tokens + already-fed answer tokens), stop step per question;
* layer stream ``default_rng([wid, 1, layer])``: raw context K, context V,
  raw segment K, segment V, in that order, ``standard_normal * value_std``;
* step stream ``default_rng([wid, 2, layer, step])``: q_new, k_new, v_new;
* prefill stream ``default_rng([wid, 3, layer])``: raw queries of every
  context token, then of every segment token (the rows of a prefill);
* two-level batches: instruction lengths from ``default_rng([wid, 4])``,
  raw instruction K then V from ``default_rng([wid, 5, layer])``.

Values are drawn as float32; bf16 workloads are then rounded to the nearest
bf16 value (ties to even) and kept as float32 arrays holding bf16 values.
Uniform integer ranges are inclusive at both ends.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Optional, Tuple

import numpy as np

__all__ = [
    "DecodeWorkload",
    "WORKLOADS",
    "workload",
    "Structure",
    "make_structure",
    "layer_kv",
    "step_inputs",
    "prefill_queries",
    "instructions",
    "round_to_bf16",
    "bf16_bits",
]


def round_to_bf16(x: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bfloat16 (ties to even), returned as float32."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    return u.astype(np.uint32).view(np.float32).reshape(x.shape)


def bf16_bits(x: np.ndarray) -> np.ndarray:
    """Upper 16 bits of float32 values that are exactly representable in bf16."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    return (x.view(np.uint32) >> 16).astype(np.uint16)


@dataclass(frozen=True)
class DecodeWorkload:
    """Shape and distribution recipe of one decode-attention workload."""

    wid: int                      # workload id, first seed word
    name: str
    dtype: str                    # "f32" or "bf16": storage / operand precision
    num_prompts: int              # B stacked prompts, each with its own context
    hq: int                       # query heads
    hkv: int                      # key/value heads
    head_dim: int                 # D
    ctx_len: Tuple[int, int]      # context tokens per prompt, inclusive range
    questions: Tuple[int, int]    # questions per prompt, inclusive range
    question_tokens: int          # fixed question part of a segment (0 -> seg_len only)
    seg_len: Tuple[int, int]      # initial segment length if question_tokens == 0,
                                  # else already-fed answer tokens range
    steps: int                    # decode steps
    layers: int = 1               # independent per-layer KV caches
    stop: Optional[Tuple[int, int]] = None   # per-question stop step range; None = all active
    value_std: float = 0.5
    rope_base: float = 10000.0

    @property
    def group(self) -> int:
        return self.hq // self.hkv

    @property
    def elem_bytes(self) -> int:
        return 4 if self.dtype == "f32" else 2


WORKLOADS = {
    # Tiny fp32 step: one prompt, Lc 256, 4 questions of 16 question + 8 answer tokens.
    1: DecodeWorkload(1, "tiny-f32", "f32", 1, 4, 2, 64, (256, 256), (4, 4), 16, (8, 8),
                      steps=1, value_std=1.0),
    # Llama-3-8B-shaped single layer, Lc 4096, 16 questions, 32 + U{0..64} tokens, 64 steps.
    2: DecodeWorkload(2, "llama3-8b-lc4096-n16", "bf16", 1, 32, 8, 128, (4096, 4096), (16, 16),
                      32, (0, 64), steps=64),
    # 32 ragged prompts: Lc U{1024..8192}, N U{4..32}, segments U{16..96}, 32 steps.
    3: DecodeWorkload(3, "ragged-b32", "bf16", 32, 32, 8, 128, (1024, 8192), (4, 32),
                      0, (16, 96), steps=32),
    # Long shared context: Lc 32768, 64 questions, segments U{16..128}, 32 steps.
    4: DecodeWorkload(4, "long-lc32768-n64", "bf16", 1, 32, 8, 128, (32768, 32768), (64, 64),
                      0, (16, 128), steps=32),
    # 32 layers, 8 prompts of Lc 8192 x 32 questions, 128 steps, stop U{16..128}.
    5: DecodeWorkload(5, "32layer-b8-lc8192-n32", "bf16", 8, 32, 8, 128, (8192, 8192), (32, 32),
                      32, (0, 0), steps=128, layers=32, stop=(16, 128)),
}


def workload(wid: int) -> DecodeWorkload:
    return WORKLOADS[wid]


@dataclass
class Structure:
    """Ragged token structure shared by all layers of a workload."""

    wl: DecodeWorkload
    ctx_len: np.ndarray           # [B] int64
    q_count: np.ndarray           # [B] int64
    seg_len0: np.ndarray          # [Nt] int64, segment length before step 0
    stop: np.ndarray              # [Nt] int64, question active at steps s < stop[i]
    q_start: np.ndarray = field(init=False)    # [B+1] CSR offsets into questions
    ctx_start: np.ndarray = field(init=False)  # [B+1] packed offsets of raw context tokens
    seg_start: np.ndarray = field(init=False)  # [Nt+1] packed offsets of raw segment tokens
    prompt_of: np.ndarray = field(init=False)  # [Nt] prompt index of each question

    def __post_init__(self):
        self.q_start = np.concatenate([[0], np.cumsum(self.q_count)]).astype(np.int64)
        self.ctx_start = np.concatenate([[0], np.cumsum(self.ctx_len)]).astype(np.int64)
        self.seg_start = np.concatenate([[0], np.cumsum(self.seg_len0)]).astype(np.int64)
        self.prompt_of = np.repeat(np.arange(len(self.q_count)), self.q_count).astype(np.int64)

    @property
    def num_questions(self) -> int:
        return int(self.q_start[-1])

    def active(self, step: int) -> np.ndarray:
        """[Nt] bool: questions still decoding at ``step`` (0-based)."""
        return step < self.stop

    def seg_len_at(self, step: int) -> np.ndarray:
        """Segment length of each question at the start of ``step`` (before its append)."""
        return self.seg_len0 + np.minimum(step, self.stop)


def make_structure(wl: DecodeWorkload) -> Structure:
    rng = np.random.default_rng([wl.wid, 0])
    B = wl.num_prompts
    ctx_len = rng.integers(wl.ctx_len[0], wl.ctx_len[1], size=B, endpoint=True)
    q_count = rng.integers(wl.questions[0], wl.questions[1], size=B, endpoint=True)
    nt = int(q_count.sum())
    fed = rng.integers(wl.seg_len[0], wl.seg_len[1], size=nt, endpoint=True)
    seg_len0 = wl.question_tokens + fed
    if wl.stop is None:
        stop = np.full(nt, wl.steps, dtype=np.int64)
    else:
        stop = rng.integers(wl.stop[0], wl.stop[1], size=nt, endpoint=True)
    return Structure(wl, ctx_len.astype(np.int64), q_count.astype(np.int64),
                     seg_len0.astype(np.int64), stop.astype(np.int64))


def _draw(rng: np.random.Generator, shape, wl: DecodeWorkload) -> np.ndarray:
    x = rng.standard_normal(size=shape, dtype=np.float32)
    if wl.value_std != 1.0:
        x *= np.float32(wl.value_std)
    if wl.dtype == "bf16":
        x = round_to_bf16(x)
    return x


@dataclass
class LayerKV:
    """Raw per-layer KV of one workload (token-major, packed, pre-rotation)."""

    ctx_k: np.ndarray   # [sum Lc, Hkv, D]
    ctx_v: np.ndarray   # [sum Lc, Hkv, D]
    seg_k: np.ndarray   # [sum seg_len0, Hkv, D]
    seg_v: np.ndarray   # [sum seg_len0, Hkv, D]


def layer_kv(st: Structure, layer: int = 0) -> LayerKV:
    wl = st.wl
    rng = np.random.default_rng([wl.wid, 1, layer])
    nc = int(st.ctx_start[-1])
    ns = int(st.seg_start[-1])
    shape_c = (nc, wl.hkv, wl.head_dim)
    shape_s = (ns, wl.hkv, wl.head_dim)
    ck = _draw(rng, shape_c, wl)
    cv = _draw(rng, shape_c, wl)
    sk = _draw(rng, shape_s, wl)
    sv = _draw(rng, shape_s, wl)
    return LayerKV(ck, cv, sk, sv)


@dataclass
class StepInputs:
    q_new: np.ndarray   # [Nt, Hq, D]  raw (pre-rotation) query of the token fed this step
    k_new: np.ndarray   # [Nt, Hkv, D] raw key of that token
    v_new: np.ndarray   # [Nt, Hkv, D]
    active: np.ndarray  # [Nt] bool


def step_inputs(st: Structure, step: int, layer: int = 0) -> StepInputs:
    wl = st.wl
    rng = np.random.default_rng([wl.wid, 2, layer, step])
    nt = st.num_questions
    q = _draw(rng, (nt, wl.hq, wl.head_dim), wl)
    k = _draw(rng, (nt, wl.hkv, wl.head_dim), wl)
    v = _draw(rng, (nt, wl.hkv, wl.head_dim), wl)
    return StepInputs(q, k, v, st.active(step))


def custom_workload(**kw) -> DecodeWorkload:
    """A workload with explicit fields (tests use it for small ragged cases)."""
    base = dict(wid=100, name="custom", dtype="f32", num_prompts=1, hq=4, hkv=2, head_dim=64,
                ctx_len=(16, 16), questions=(2, 2), question_tokens=0, seg_len=(4, 4),
                steps=1)
    base.update(kw)
    return DecodeWorkload(**base)


@dataclass
class PrefillQueries:
    ctx_q: np.ndarray   # [sum Lc, Hq, D]        raw queries of the context tokens
    seg_q: np.ndarray   # [sum seg_len0, Hq, D]  raw queries of the segment tokens


def prefill_queries(st: Structure, layer: int = 0) -> PrefillQueries:
    """Raw query vectors of every token of the stacked header (prefill rows)."""
    wl = st.wl
    rng = np.random.default_rng([wl.wid, 3, layer])
    cq = _draw(rng, (int(st.ctx_start[-1]), wl.hq, wl.head_dim), wl)
    sq = _draw(rng, (int(st.seg_start[-1]), wl.hq, wl.head_dim), wl)
    return PrefillQueries(cq, sq)


@dataclass
class InstructionKV:
    """Instruction blocks of a two-level batch: prompts prompt_start[s] ..
    prompt_start[s+1]-1 sit behind instruction s of lp[s] tokens, whose raw
    keys/values are k/v[tok_start[s]:tok_start[s+1]]."""

    prompt_start: np.ndarray   # [S+1]
    lp: np.ndarray             # [S]
    tok_start: np.ndarray      # [S+1]
    k: np.ndarray              # [sum lp, Hkv, D]
    v: np.ndarray


def instructions(st: Structure, contexts_per_instr: int, lp: Tuple[int, int], layer: int = 0) -> InstructionKV:
    """Consecutive prompts grouped contexts_per_instr at a time (the last group
    may be smaller) behind instructions of U{lp} tokens."""
    wl = st.wl
    B = wl.num_prompts
    prompt_start = np.array(list(range(0, B, contexts_per_instr)) + [B], dtype=np.int64)
    S = len(prompt_start) - 1
    lens = np.random.default_rng([wl.wid, 4]).integers(lp[0], lp[1], size=S, endpoint=True).astype(np.int64)
    tok_start = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    rng = np.random.default_rng([wl.wid, 5, layer])
    shape = (int(tok_start[-1]), wl.hkv, wl.head_dim)
    k = _draw(rng, shape, wl)
    v = _draw(rng, shape, wl)
    return InstructionKV(prompt_start, lens, tok_start, k, v)


def instruction_queries(st: Structure, ins: InstructionKV, layer: int = 0) -> np.ndarray:
    """Raw query vectors of every instruction token (prefill rows), [sum lp, Hq, D]."""
    wl = st.wl
    rng = np.random.default_rng([wl.wid, 6, layer])
    return _draw(rng, (int(ins.tok_start[-1]), wl.hq, wl.head_dim), wl)
