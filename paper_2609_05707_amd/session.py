"""Torch-side buffers for one batch of stacked prompts, wired to the C ABI.

PyTorch only provides device memory and the stream here.  A DecodeBatch
owns, per emulated layer, the KV cache of the library layout and the
segment-length counters; it fills ``ippd_batch_t`` / ``ippd_kv_cache_t``
structs and forwards every operation to libippd.
"""
from __future__ import annotations

from typing import Optional, Sequence

import numpy as np
import torch

from . import _lib as L


def _round8(x: int) -> int:
    return (int(x) + 7) // 8 * 8


def torch_dtype(dtype: str):
    return torch.float32 if dtype == "f32" else torch.bfloat16


class DecodeBatch:
    """B prompts (context lengths ``ctx_len``, question counts ``q_count``) on one GPU.

    Context pool: prompt b at token offset ctx_off[b] (multiples of 8, packed).
    ``layers`` independent caches share the structure arrays and the active
    mask; each layer has its own seg_len counters (advanced by its appends).
    """

    def __init__(self, ctx_len: Sequence[int], q_count: Sequence[int], hq: int, hkv: int,
                 head_dim: int, dtype: str, seg_capacity: int, rope_base: float = 10000.0,
                 scale: float = 0.0, chunk_tokens: int = 0, max_questions: Optional[int] = None,
                 layers: int = 1, tile_rows: int = 0, device: str = "cuda",
                 instr_len: Optional[Sequence[int]] = None, instr_prompt_start: Optional[Sequence[int]] = None):
        """instr_len / instr_prompt_start (optional) make a two-level batch:
        prompts instr_prompt_start[s] .. instr_prompt_start[s+1]-1 sit behind
        instruction s of instr_len[s] tokens, held at the front of the pool."""
        self.device = torch.device(device)
        self.dtype = dtype
        self.tdtype = torch_dtype(dtype)
        self.B = len(ctx_len)
        self.ctx_len = np.asarray(ctx_len, dtype=np.int64)
        self.q_count = np.asarray(q_count, dtype=np.int64)
        self.Nt = int(self.q_count.sum())
        self.hq, self.hkv, self.D = hq, hkv, head_dim
        self.seg_cap = _round8(max(seg_capacity, 8))
        self.layers = layers
        self.S = 0 if instr_len is None else len(instr_len)
        self.instr_len = np.asarray(instr_len if instr_len is not None else [], dtype=np.int64)
        ipad = np.array([_round8(x) for x in self.instr_len], dtype=np.int64)
        self.instr_off = np.concatenate([[0], np.cumsum(ipad)[:-1]]).astype(np.int64) if self.S else ipad
        ibase = int(ipad.sum())
        padded = np.array([_round8(x) for x in self.ctx_len], dtype=np.int64)
        self.ctx_off = ibase + np.concatenate([[0], np.cumsum(padded)[:-1]]).astype(np.int64)
        self.pool = max(8, ibase + int(padded.sum()))
        self.q_start = np.concatenate([[0], np.cumsum(self.q_count)]).astype(np.int32)
        self.max_ctx_len = int(self.ctx_len.max()) if self.B else 0
        self.max_questions = int(max_questions if max_questions is not None
                                 else max(1, int(self.q_count.max())))
        dev = self.device
        self.d_ctx_off = torch.from_numpy(self.ctx_off).to(dev)
        self.d_ctx_len = torch.from_numpy(self.ctx_len.astype(np.int32)).to(dev)
        self.d_q_start = torch.from_numpy(self.q_start).to(dev)
        self.d_active = torch.ones(max(self.Nt, 1), dtype=torch.uint8, device=dev)
        self.d_err = torch.zeros(1, dtype=torch.int32, device=dev)
        if self.S:
            self.instr_prompt_start = np.asarray(instr_prompt_start, dtype=np.int32)
            if len(self.instr_prompt_start) != self.S + 1:
                raise ValueError("instr_prompt_start needs num_instr + 1 entries")
            self.max_instr_questions = max(1, max(int(self.q_start[self.instr_prompt_start[s + 1]] -
                                                      self.q_start[self.instr_prompt_start[s]])
                                                  for s in range(self.S)))
            self.d_instr_start = torch.from_numpy(self.instr_prompt_start).to(dev)
            self.d_instr_off = torch.from_numpy(self.instr_off).to(dev)
            self.d_instr_len = torch.from_numpy(self.instr_len.astype(np.int32)).to(dev)
        self.seg_len = [torch.zeros(max(self.Nt, 1), dtype=torch.int32, device=dev) for _ in range(layers)]
        td = self.tdtype
        self.ctx_k = [torch.empty(hkv, self.pool, head_dim, dtype=td, device=dev) for _ in range(layers)]
        # values transposed in 8-token column blocks (see include/ippd.h)
        self.ctx_vt = [torch.empty(hkv, self.pool // 8, head_dim, 8, dtype=td, device=dev) for _ in range(layers)]
        nt = max(self.Nt, 1)
        self.seg_k = [torch.empty(nt, hkv, self.seg_cap, head_dim, dtype=td, device=dev) for _ in range(layers)]
        self.seg_vt = [torch.empty(nt, hkv, self.seg_cap // 8, head_dim, 8, dtype=td, device=dev)
                       for _ in range(layers)]
        self.batches = []
        self.caches = []
        for layer in range(layers):
            bt = L.IppdBatch()
            bt.num_prompts = self.B
            bt.num_questions = self.Nt
            bt.num_q_heads = hq
            bt.num_kv_heads = hkv
            bt.head_dim = head_dim
            bt.dtype = L.IPPD_DTYPE_F32 if dtype == "f32" else L.IPPD_DTYPE_BF16
            bt.ctx_pool_tokens = self.pool
            bt.seg_capacity = self.seg_cap
            bt.max_ctx_len = self.max_ctx_len
            bt.max_questions = self.max_questions
            bt.chunk_tokens = chunk_tokens
            bt.tile_rows = tile_rows
            bt.rope_base = rope_base
            bt.scale = scale
            bt.ctx_off = self.d_ctx_off.data_ptr()
            bt.ctx_len = self.d_ctx_len.data_ptr()
            bt.q_start = self.d_q_start.data_ptr()
            bt.seg_len = self.seg_len[layer].data_ptr()
            bt.active = self.d_active.data_ptr()
            bt.err_flag = self.d_err.data_ptr()
            if self.S:
                bt.num_instr = self.S
                bt.max_instr_len = int(self.instr_len.max())
                bt.max_instr_questions = self.max_instr_questions
                bt.instr_start = self.d_instr_start.data_ptr()
                bt.instr_off = self.d_instr_off.data_ptr()
                bt.instr_len = self.d_instr_len.data_ptr()
            self.batches.append(bt)
            kv = L.IppdKvCache()
            kv.ctx_k = self.ctx_k[layer].data_ptr()
            kv.ctx_vt = self.ctx_vt[layer].data_ptr()
            kv.seg_k = self.seg_k[layer].data_ptr()
            kv.seg_vt = self.seg_vt[layer].data_ptr()
            self.caches.append(kv)
        self.ws_dense_bytes = L.dense_decode_workspace_bytes(self.batches[0])   # 0 if not supported
        self.ws_ippd_bytes = L.ippd_decode_workspace_bytes(self.batches[0])
        self.ws_std_bytes = L.standard_decode_workspace_bytes(self.batches[0])
        # the library needs no initialisation of its workspace (zeros for tidiness)
        self.ws_ippd = torch.zeros(max(self.ws_ippd_bytes, 256), dtype=torch.uint8, device=dev)
        self.ws_std = torch.zeros(max(self.ws_std_bytes, 256), dtype=torch.uint8, device=dev)
        self.q_rot = torch.empty(nt, hq, head_dim, dtype=td, device=dev)
        self.out = torch.empty(nt, hq, head_dim, dtype=torch.float32, device=dev)
        self.lse = torch.empty(nt, hq, dtype=torch.float32, device=dev)

    # ------------------------------------------------------------------ helpers
    @staticmethod
    def stream() -> int:
        return torch.cuda.current_stream().cuda_stream

    def to_dev(self, x) -> torch.Tensor:
        t = x if isinstance(x, torch.Tensor) else torch.from_numpy(np.ascontiguousarray(x))
        return t.to(self.device).to(self.tdtype).contiguous()

    def ctx_values(self, layer: int) -> torch.Tensor:
        """Context values of one layer as [Hkv][D][pool] (a copy; the cache holds
        them in 8-token column blocks)."""
        x = self.ctx_vt[layer]
        return x.permute(0, 2, 1, 3).reshape(self.hkv, self.D, self.pool)

    def seg_values(self, layer: int) -> torch.Tensor:
        """Segment values of one layer as [Nt][Hkv][D][seg_capacity] (a copy)."""
        x = self.seg_vt[layer]
        return x.permute(0, 1, 3, 2, 4).reshape(x.shape[0], self.hkv, self.D, self.seg_cap)

    def err_flag(self) -> int:
        return int(self.d_err.item())

    # ------------------------------------------------------------------ loading
    def load_context(self, layer: int, k_packed, v_packed) -> None:
        """k/v_packed: [sum ctx_len, Hkv, D] raw (pre-rotation), prompts in order."""
        kp, vp = self.to_dev(k_packed), self.to_dev(v_packed)
        k_raw = torch.zeros(self.pool, self.hkv, self.D, dtype=self.tdtype, device=self.device)
        v_raw = torch.zeros_like(k_raw)
        src = 0
        for b in range(self.B):
            n = int(self.ctx_len[b])
            o = int(self.ctx_off[b])
            k_raw[o:o + n] = kp[src:src + n]
            v_raw[o:o + n] = vp[src:src + n]
            src += n
        L.ippd_load_context(self.batches[layer], k_raw.data_ptr(), v_raw.data_ptr(),
                            self.caches[layer], self.stream())
        torch.cuda.current_stream().synchronize()

    def load_instructions(self, layer: int, k_packed, v_packed) -> None:
        """k/v_packed: [sum instr_len, Hkv, D] raw (pre-rotation), instructions in order."""
        kp, vp = self.to_dev(k_packed), self.to_dev(v_packed)
        k_raw = torch.zeros(self.pool, self.hkv, self.D, dtype=self.tdtype, device=self.device)
        v_raw = torch.zeros_like(k_raw)
        src = 0
        for s in range(self.S):
            n, o = int(self.instr_len[s]), int(self.instr_off[s])
            k_raw[o:o + n] = kp[src:src + n]
            v_raw[o:o + n] = vp[src:src + n]
            src += n
        L.ippd_load_instructions(self.batches[layer], k_raw.data_ptr(), v_raw.data_ptr(),
                                 self.caches[layer], self.stream())
        torch.cuda.current_stream().synchronize()

    def load_segments(self, layer: int, k_packed, v_packed, seg_len0) -> None:
        """k/v_packed: [sum seg_len0, Hkv, D] raw; question i owns the next seg_len0[i] rows."""
        seg_len0 = np.asarray(seg_len0, dtype=np.int64)
        if self.Nt == 0:
            return                                      # a batch without questions has no segments
        if int(seg_len0.max()) > self.seg_cap:
            raise ValueError("initial segment longer than seg_capacity")
        kp, vp = self.to_dev(k_packed), self.to_dev(v_packed)
        nt = max(self.Nt, 1)
        k_raw = torch.zeros(nt, self.seg_cap, self.hkv, self.D, dtype=self.tdtype, device=self.device)
        v_raw = torch.zeros_like(k_raw)
        starts = np.concatenate([[0], np.cumsum(seg_len0)])
        for i in range(self.Nt):
            n = int(seg_len0[i])
            k_raw[i, :n] = kp[starts[i]:starts[i] + n]
            v_raw[i, :n] = vp[starts[i]:starts[i] + n]
        init = torch.from_numpy(seg_len0.astype(np.int32)).to(self.device)
        L.ippd_load_segments(self.batches[layer], k_raw.data_ptr(), v_raw.data_ptr(), init.data_ptr(),
                             self.caches[layer], self.stream())
        torch.cuda.current_stream().synchronize()

    def set_active(self, mask) -> None:
        m = torch.as_tensor(np.asarray(mask, dtype=np.uint8))
        self.d_active[: self.Nt].copy_(m.to(self.device))

    # ------------------------------------------------------------------ hot path
    def append(self, layer: int, q_new: torch.Tensor, k_new: torch.Tensor, v_new: torch.Tensor,
               q_rot: Optional[torch.Tensor] = None) -> None:
        q_rot = self.q_rot if q_rot is None else q_rot
        L.ippd_append_kv(self.batches[layer], q_new.data_ptr(), k_new.data_ptr(), v_new.data_ptr(),
                         q_rot.data_ptr(), self.caches[layer], self.stream())

    def decode(self, layer: int, standard: bool = False, q_rot: Optional[torch.Tensor] = None,
               out: Optional[torch.Tensor] = None, lse: Optional[torch.Tensor] = None,
               with_lse: bool = True, dense: bool = False) -> None:
        """Attention after append: IPPD, the standard baseline or (dense=True) the
        dense-mask baseline."""
        q_rot = self.q_rot if q_rot is None else q_rot
        out = self.out if out is None else out
        lse = self.lse if lse is None else lse
        lse_ptr = lse.data_ptr() if with_lse else None
        if dense:
            if self.ws_dense_bytes == 0:
                raise ValueError("the dense-mask baseline needs a one-level batch with <= 64 questions per prompt")
            if getattr(self, "ws_dense", None) is None:
                self.ws_dense = torch.zeros(self.ws_dense_bytes, dtype=torch.uint8, device=self.device)
            L.dense_decode_attention(self.batches[layer], q_rot.data_ptr(), self.caches[layer], out.data_ptr(),
                                     lse_ptr, self.ws_dense.data_ptr(), self.ws_dense_bytes, self.stream())
        elif standard:
            L.standard_decode_attention(self.batches[layer], q_rot.data_ptr(), self.caches[layer],
                                        out.data_ptr(), lse_ptr, self.ws_std.data_ptr(),
                                        self.ws_std_bytes, self.stream())
        else:
            L.ippd_decode_attention(self.batches[layer], q_rot.data_ptr(), self.caches[layer],
                                    out.data_ptr(), lse_ptr, self.ws_ippd.data_ptr(),
                                    self.ws_ippd_bytes, self.stream())

    def decode_step(self, layer: int, q_new: torch.Tensor, k_new: torch.Tensor, v_new: torch.Tensor,
                    standard: bool = False, q_rot: Optional[torch.Tensor] = None,
                    out: Optional[torch.Tensor] = None, lse: Optional[torch.Tensor] = None,
                    write_q_rot: bool = True, with_lse: bool = True) -> None:
        """Fused step: rotate + append + attention in one launch."""
        q_rot = self.q_rot if q_rot is None else q_rot
        out = self.out if out is None else out
        lse = self.lse if lse is None else lse
        qr = q_rot.data_ptr() if write_q_rot else None
        lse_ptr = lse.data_ptr() if with_lse else None
        fn = L.standard_decode_step if standard else L.ippd_decode_step
        ws, wsb = (self.ws_std, self.ws_std_bytes) if standard else (self.ws_ippd, self.ws_ippd_bytes)
        fn(self.batches[layer], q_new.data_ptr(), k_new.data_ptr(), v_new.data_ptr(), qr, self.caches[layer],
           out.data_ptr(), lse_ptr, ws.data_ptr(), wsb, self.stream())

    # ------------------------------------------------------------------ prefill
    def pack_prefill_queries(self, ctx_q, seg_q, seg_len0, instr_q=None):
        """Raw prefill queries in the library layouts: q_ctx [pool][Hq][D] (prompt
        b's context token t at row ctx_off[b] + t, instruction s's token t at
        instr_off[s] + t) and q_seg [Nt][seg_capacity][Hq][D] (question i's token
        u at [i][u]).  ctx_q [sum Lc, Hq, D], seg_q [sum seg_len0, Hq, D] and
        instr_q [sum instr_len, Hq, D] are packed in prompt / question /
        instruction order."""
        if self.S and instr_q is None:
            raise ValueError("a two-level batch needs the instruction queries (instr_q)")
        cq, sq = self.to_dev(ctx_q), self.to_dev(seg_q)
        q_ctx = torch.zeros(self.pool, self.hq, self.D, dtype=self.tdtype, device=self.device)
        src = 0
        for b in range(self.B):
            n, o = int(self.ctx_len[b]), int(self.ctx_off[b])
            q_ctx[o:o + n] = cq[src:src + n]
            src += n
        if self.S:
            iq = self.to_dev(instr_q)
            src = 0
            for s_ in range(self.S):
                n, o = int(self.instr_len[s_]), int(self.instr_off[s_])
                q_ctx[o:o + n] = iq[src:src + n]
                src += n
        nt = max(self.Nt, 1)
        q_seg = torch.zeros(nt, self.seg_cap, self.hq, self.D, dtype=self.tdtype, device=self.device)
        starts = np.concatenate([[0], np.cumsum(np.asarray(seg_len0, dtype=np.int64))])
        for i in range(self.Nt):
            n = int(starts[i + 1] - starts[i])
            q_seg[i, :n] = sq[starts[i]:starts[i] + n]
        return q_ctx, q_seg

    def prefill_outputs(self, fill: float = 0.0):
        """float32 out_ctx [pool][Hq][D] and out_seg [Nt][seg_capacity][Hq][D]."""
        nt = max(self.Nt, 1)
        oc = torch.full((self.pool, self.hq, self.D), fill, dtype=torch.float32, device=self.device)
        os_ = torch.full((nt, self.seg_cap, self.hq, self.D), fill, dtype=torch.float32, device=self.device)
        return oc, os_

    def prefill(self, layer: int, q_ctx: torch.Tensor, q_seg: torch.Tensor, out_ctx: torch.Tensor,
                out_seg: torch.Tensor, max_prompt_question_tokens: int, standard: bool = False) -> None:
        """Prefill attention of every instruction, context and question token (the
        segments hold the question tokens: load them with load_segments first)."""
        fn = L.standard_prefill_attention if standard else L.ippd_prefill_attention
        fn(self.batches[layer], int(max_prompt_question_tokens), q_ctx.data_ptr(), q_seg.data_ptr(),
           self.caches[layer], out_ctx.data_ptr(), out_seg.data_ptr(), self.stream())
