"""C ABI checks that need no GPU: the library loads, exports every entry point
declared in include/ippd.h, and rejects bad arguments on the host before any
launch (so no device memory is touched by these calls)."""
import ctypes
import os
import re

import pytest

from paper_2609_05707_amd import _lib as L

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "ippd.h")

# Fake, never-dereferenced device addresses (validation fails before any launch).
FAKE = 0x10000
MISALIGNED = 0x10008 + 1


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    names = re.findall(r"^\s*(?:const\s+)?[a-z_0-9]+\s*\*?\s*([a-z_0-9]+)\s*\(", src, flags=re.M)
    return sorted(set(names))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(L.LIB_PATH):
        pytest.fail("libippd.so not built (run __graft_entry__.build())")
    return L.load_library()


def test_exports_every_declared_symbol(lib):
    names = declared_functions()
    assert set(names) == set(L.EXPORTED), names
    for n in names:
        assert hasattr(lib, n), n


def valid_batch(**kw):
    bt = L.IppdBatch()
    bt.num_prompts, bt.num_questions, bt.num_q_heads, bt.num_kv_heads = 1, 4, 4, 2
    bt.head_dim, bt.dtype = 64, L.IPPD_DTYPE_F32
    bt.ctx_pool_tokens, bt.seg_capacity, bt.max_ctx_len, bt.max_questions = 256, 32, 256, 4
    bt.chunk_tokens, bt.tile_rows, bt.rope_base, bt.scale = 0, 0, 10000.0, 0.0
    for f in ("ctx_off", "ctx_len", "q_start", "seg_len", "active", "err_flag"):
        setattr(bt, f, FAKE)
    for k, v in kw.items():
        setattr(bt, k, v)
    return bt


def kv_cache(ptr=FAKE):
    kv = L.IppdKvCache()
    kv.ctx_k = kv.ctx_vt = kv.seg_k = kv.seg_vt = ptr
    return kv


def decode_status(lib, bt, q=FAKE, out=FAKE, ws=FAKE, ws_bytes=None, kv=None, fn="ippd_decode_attention"):
    if ws_bytes is None:
        ws_bytes = 1 << 30
    return getattr(lib, fn)(ctypes.byref(bt), q, ctypes.byref(kv or kv_cache()), out, None, ws,
                            ws_bytes, None)


def test_version_and_strings(lib):
    assert lib.ippd_version() >= 100
    for s in range(8):
        assert lib.ippd_status_string(s)
    assert lib.ippd_last_hip_error() == 0


@pytest.mark.parametrize("field,value,status", [
    ("num_kv_heads", 3, L.IPPD_ERR_SHAPE),          # Hq % Hkv != 0
    ("head_dim", 96, L.IPPD_ERR_SHAPE),
    ("dtype", 7, L.IPPD_ERR_DTYPE),
    ("ctx_pool_tokens", 250, L.IPPD_ERR_SHAPE),     # not a multiple of 8
    ("seg_capacity", 12, L.IPPD_ERR_SHAPE),
    ("max_ctx_len", 300, L.IPPD_ERR_SHAPE),         # beyond the pool
    ("max_questions", 0, L.IPPD_ERR_SHAPE),
    ("max_questions", 2000, L.IPPD_ERR_SHAPE),
    ("chunk_tokens", 48, L.IPPD_ERR_SHAPE),         # not a multiple of 32
    ("tile_rows", 24, L.IPPD_ERR_SHAPE),
    ("tile_rows", 256, L.IPPD_ERR_SHAPE),
    ("num_q_heads", 68, L.IPPD_ERR_SHAPE),          # 34 query heads per kv head
    ("rope_base", -1.0, L.IPPD_ERR_SHAPE),
    ("num_prompts", 0, L.IPPD_ERR_SHAPE),
    ("seg_len", None, L.IPPD_ERR_NULL),
    ("err_flag", None, L.IPPD_ERR_NULL),
])
def test_batch_validation(lib, field, value, status):
    bt = valid_batch(**{field: value})
    assert decode_status(lib, bt) == status
    assert lib.ippd_append_kv(ctypes.byref(bt), FAKE, FAKE, FAKE, FAKE, ctypes.byref(kv_cache()), None) == status
    assert lib.ippd_decode_workspace_bytes(ctypes.byref(bt)) == 0
    for fn in ("ippd_prefill_attention", "standard_prefill_attention"):
        assert getattr(lib, fn)(ctypes.byref(bt), 8, FAKE, FAKE, ctypes.byref(kv_cache()), FAKE, FAKE,
                                None) == status


def test_pointer_validation(lib):
    bt = valid_batch()
    assert decode_status(lib, bt, q=None) == L.IPPD_ERR_NULL
    assert decode_status(lib, bt, out=None) == L.IPPD_ERR_NULL
    assert decode_status(lib, bt, kv=kv_cache(0)) == L.IPPD_ERR_NULL
    assert decode_status(lib, bt, q=MISALIGNED) == L.IPPD_ERR_ALIGN
    assert decode_status(lib, bt, kv=kv_cache(MISALIGNED)) == L.IPPD_ERR_ALIGN
    assert lib.ippd_append_kv(ctypes.byref(bt), MISALIGNED, FAKE, FAKE, FAKE,
                              ctypes.byref(kv_cache()), None) == L.IPPD_ERR_ALIGN
    assert lib.ippd_load_context(ctypes.byref(bt), None, FAKE, ctypes.byref(kv_cache()), None) == L.IPPD_ERR_NULL
    assert lib.ippd_load_segments(ctypes.byref(bt), FAKE, FAKE, None, ctypes.byref(kv_cache()),
                                  None) == L.IPPD_ERR_NULL
    assert lib.ippd_decode_attention(None, FAKE, ctypes.byref(kv_cache()), FAKE, None, FAKE, 1, None) \
        == L.IPPD_ERR_NULL


def test_workspace_validation(lib):
    bt = valid_batch()
    need = lib.ippd_decode_workspace_bytes(ctypes.byref(bt))
    need_std = lib.standard_decode_workspace_bytes(ctypes.byref(bt))
    assert need > 0 and need_std > 0
    assert decode_status(lib, bt, ws_bytes=need - 1) == L.IPPD_ERR_WORKSPACE
    assert decode_status(lib, bt, ws=None) == L.IPPD_ERR_WORKSPACE
    assert decode_status(lib, bt, ws=FAKE + 16, ws_bytes=need) == L.IPPD_ERR_ALIGN
    assert decode_status(lib, bt, ws_bytes=need_std - 1, fn="standard_decode_attention") == \
        L.IPPD_ERR_WORKSPACE


def test_workspace_formula(lib):
    # (max_chunks + 1) * Nt * Hq partial states of D + 2 floats (chunks, then
    # the segment), each array 256-byte rounded.  Both modes alike.
    bt = valid_batch(chunk_tokens=64)
    slots = (256 // 64 + 1) * 4 * 4
    r = lambda x: (x + 255) // 256 * 256
    want = r(slots * 64 * 4) + r(slots * 2 * 4)
    assert lib.ippd_decode_workspace_bytes(ctypes.byref(bt)) == want
    assert lib.standard_decode_workspace_bytes(ctypes.byref(bt)) == want


def test_step_pointer_validation(lib):
    bt = valid_batch()
    kv = kv_cache()
    args = lambda q, k, v: (ctypes.byref(bt), q, k, v, None, ctypes.byref(kv), FAKE, None, FAKE, 1 << 30, None)
    assert lib.ippd_decode_step(*args(None, FAKE, FAKE)) == L.IPPD_ERR_NULL
    assert lib.standard_decode_step(*args(FAKE, None, FAKE)) == L.IPPD_ERR_NULL
    assert lib.ippd_decode_step(*args(FAKE, FAKE, MISALIGNED)) == L.IPPD_ERR_ALIGN


def test_no_questions_is_a_noop(lib):
    bt = valid_batch(num_questions=0)
    assert decode_status(lib, bt, ws=None, ws_bytes=0) == L.IPPD_OK


def test_prefill_validation(lib):
    bt = valid_batch()
    for fn in ("ippd_prefill_attention", "standard_prefill_attention"):
        f = getattr(lib, fn)

        def call(m=64, qc=FAKE, qs=FAKE, oc=FAKE, os_=FAKE, kv=None):
            return f(ctypes.byref(bt), m, qc, qs, ctypes.byref(kv or kv_cache()), oc, os_, None)
        assert call(qc=None) == L.IPPD_ERR_NULL
        assert call(qs=None) == L.IPPD_ERR_NULL
        assert call(oc=None) == L.IPPD_ERR_NULL
        assert call(os_=None) == L.IPPD_ERR_NULL
        assert call(kv=kv_cache(0)) == L.IPPD_ERR_NULL
        assert call(qs=MISALIGNED) == L.IPPD_ERR_ALIGN
        assert call(oc=MISALIGNED) == L.IPPD_ERR_ALIGN
        assert call(kv=kv_cache(MISALIGNED)) == L.IPPD_ERR_ALIGN
        assert call(m=-1) == L.IPPD_ERR_SHAPE
    assert lib.ippd_version() >= 500


def test_instruction_level_validation(lib):
    kv = kv_cache()
    bad = [(dict(num_instr=-1), L.IPPD_ERR_SHAPE),
           (dict(num_instr=2), L.IPPD_ERR_SHAPE),                       # more instructions than prompts
           (dict(num_instr=1, max_instr_len=8, max_instr_questions=0), L.IPPD_ERR_SHAPE),
           (dict(num_instr=1, max_instr_len=300, max_instr_questions=4), L.IPPD_ERR_SHAPE),   # beyond the pool
           (dict(num_instr=1, max_instr_len=8, max_instr_questions=4), L.IPPD_ERR_NULL)]      # arrays missing
    for kw, status in bad:
        bt = valid_batch(**kw)
        assert decode_status(lib, bt) == status, kw
        assert lib.ippd_load_instructions(ctypes.byref(bt), FAKE, FAKE, ctypes.byref(kv), None) == status, kw
        for fn in (lib.ippd_prefill_attention, lib.standard_prefill_attention):
            assert fn(ctypes.byref(bt), 8, FAKE, FAKE, ctypes.byref(kv), FAKE, FAKE, None) == status, kw
    bt = valid_batch()
    assert lib.ippd_load_instructions(ctypes.byref(bt), FAKE, FAKE, ctypes.byref(kv), None) == L.IPPD_ERR_SHAPE
    good = valid_batch(num_instr=1, max_instr_len=64, max_instr_questions=4, instr_start=FAKE, instr_off=FAKE,
                       instr_len=FAKE)
    assert lib.ippd_load_instructions(ctypes.byref(good), None, FAKE, ctypes.byref(kv), None) == L.IPPD_ERR_NULL
    # a valid two-level batch passes the prefill's checks up to its pointers (0.6.0 on)
    assert lib.ippd_version() >= 600
    assert lib.ippd_prefill_attention(ctypes.byref(good), 8, None, FAKE, ctypes.byref(kv), FAKE, FAKE,
                                      None) == L.IPPD_ERR_NULL


def test_workspace_formula_with_instructions(lib):
    # (max_chunks + 1 + max_ichunks) * Nt * Hq partial states: context chunks,
    # the segment, then instruction chunks
    bt = valid_batch(chunk_tokens=64, num_instr=1, max_instr_len=100, max_instr_questions=4, instr_start=FAKE,
                     instr_off=FAKE, instr_len=FAKE)
    slots = (256 // 64 + 1 + 2) * 4 * 4
    r = lambda x: (x + 255) // 256 * 256
    want = r(slots * 64 * 4) + r(slots * 2 * 4)
    assert lib.ippd_decode_workspace_bytes(ctypes.byref(bt)) == want
    assert lib.standard_decode_workspace_bytes(ctypes.byref(bt)) == want


def test_dense_baseline_validation(lib):
    bt = valid_batch()
    need = lib.dense_decode_workspace_bytes(ctypes.byref(bt))
    assert need >= lib.ippd_decode_workspace_bytes(ctypes.byref(bt))      # + any segment chunk slots
    assert decode_status(lib, bt, ws_bytes=need - 1, fn="dense_decode_attention") == L.IPPD_ERR_WORKSPACE
    assert decode_status(lib, bt, q=None, fn="dense_decode_attention") == L.IPPD_ERR_NULL
    many = valid_batch(max_questions=65)                                   # more than 64 questions per prompt
    assert lib.dense_decode_workspace_bytes(ctypes.byref(many)) == 0
    assert decode_status(lib, many, fn="dense_decode_attention") == L.IPPD_ERR_SHAPE
    two = valid_batch(num_instr=1, max_instr_len=64, max_instr_questions=4, instr_start=FAKE, instr_off=FAKE,
                      instr_len=FAKE)
    assert decode_status(lib, two, fn="dense_decode_attention") == L.IPPD_ERR_SHAPE


def test_noalloc_step_rejects_batches_beyond_its_scratch(lib):
    """ippd_decode_step_noalloc returns IPPD_ERR_SCRATCH, before any HIP call,
    for a batch whose partial states exceed IPPD_NOALLOC_SCRATCH_BYTES, and
    validates the batch like the other entry points."""
    assert lib.ippd_version() >= 700
    kv = kv_cache()
    # 1024 questions x 32 heads x (16 context chunks + segment) x 130 floats: far above 64 MiB
    big = valid_batch(num_questions=1024, max_questions=1024, num_q_heads=32, num_kv_heads=8, head_dim=128,
                      ctx_pool_tokens=65536, max_ctx_len=65536, chunk_tokens=4096)
    need = lib.ippd_decode_workspace_bytes(ctypes.byref(big))
    assert need > L.IPPD_NOALLOC_SCRATCH_BYTES
    assert lib.ippd_decode_step_noalloc(ctypes.byref(big), FAKE, FAKE, FAKE, FAKE, ctypes.byref(kv), FAKE, None,
                                        None) == L.IPPD_ERR_SCRATCH
    assert lib.ippd_status_string(L.IPPD_ERR_SCRATCH)
    bad = valid_batch(head_dim=96)
    assert lib.ippd_decode_step_noalloc(ctypes.byref(bad), FAKE, FAKE, FAKE, FAKE, ctypes.byref(kv), FAKE, None,
                                        None) == L.IPPD_ERR_SHAPE
    assert lib.ippd_last_hip_error() == 0
