"""CPU: the host side of bench.py.  One GPU only (--gpus above 1 exits before
touching a device), and the byte and FLOP bookkeeping behind value and the
roofline, checked by hand on a tiny ragged step: one prompt with all of its
questions active, one whose only question has stopped."""
import os
import subprocess
import sys

import numpy as np

import bench
import workload as W

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_more_than_one_gpu_exits_with_a_message():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120)
    assert r.returncode == 2
    assert "one GPU" in r.stderr


def _tiny():
    wl = W.custom_workload(wid=900, dtype="bf16", num_prompts=2, hq=8, hkv=2, head_dim=64, steps=2)
    # prompt 0: context 100, questions with 3 and 5 cached tokens (both decode at step 0);
    # prompt 1: context 50, one question with 7 tokens that has already stopped
    return W.Structure(wl, np.array([100, 50]), np.array([2, 1]), np.array([3, 5, 7]), np.array([1, 1, 0]))


def test_step_bytes_by_hand():
    st = _tiny()
    e, D, hq, hkv = 2, 64, 8, 2
    ctx0 = 2 * 100 * hkv * D * e                      # K and V of prompt 0's context; prompt 1 is idle
    segs = 2 * (3 + 5) * hkv * D * e                  # cached segment K and V of the two active questions
    per_q = (hq + 2 * hkv) * D * e + 2 * hkv * D * e + hq * D * 4 + hq * 4   # q/k/v in, k/v appended, out + lse
    assert bench.step_bytes(st, 0) == ctx0 + segs + 2 * per_q == 63552
    # the baseline reads prompt 0's context once per active question
    assert bench.step_bytes(st, 0, standard=True) == 2 * ctx0 + segs + 2 * per_q
    # step 1: every question has stopped
    assert bench.step_bytes(st, 1) == 0


def test_step_flops_by_hand():
    st = _tiny()
    # Q.K and P.V over context + cached segment + the step's own token, per query head
    expect = 4 * 8 * 64 * ((100 + 3 + 1) + (100 + 5 + 1))
    assert bench.step_flops(st, 0) == expect
    assert bench.step_flops(st, 1) == 0


def test_prefill_flops_by_hand():
    """bench_prefill's algorithmic FLOPs, 4*D*Hq per visible (row, key) pair: one
    prompt (context 10, questions of 3 and 4 tokens), then behind an instruction
    of 5 tokens."""
    import bench_prefill as BP
    wl = W.custom_workload(wid=901, dtype="bf16", num_prompts=1, hq=8, hkv=2, head_dim=64, steps=1)
    st = W.Structure(wl, np.array([10]), np.array([2]), np.array([3, 4]), np.array([1, 1]))
    per = 4 * 64 * 8
    ctx = 10 * 11 // 2                                  # causal context rows
    q = (3 * 10 + 3 * 4 // 2) + (4 * 10 + 4 * 5 // 2)   # whole context + causal own question
    assert BP.flops(st, False) == per * (ctx + q)
    assert BP.flops(st, True) == per * (2 * ctx + q)   # the context rows once per question
    ins = W.InstructionKV(np.array([0, 1]), np.array([5]), np.array([0, 5]), None, None)
    ins_rows = 5 * 6 // 2
    ctx_i = 10 * 5 + ctx                                # every context row also sees the instruction
    q_i = (3 * 15 + 3 * 4 // 2) + (4 * 15 + 4 * 5 // 2)
    assert BP.flops(st, False, ins) == per * (ins_rows + ctx_i + q_i)
    assert BP.flops(st, True, ins) == per * (2 * ins_rows + 2 * ctx_i + q_i)


def test_counter_fingerprint_ignores_comments_but_not_code(tmp_path):
    """A counter record stays valid across comment and layout edits of the
    kernel sources, and not across a code change."""
    import shutil
    from paper_2609_05707_amd import traffic as T
    src = os.path.join(ROOT, "paper_2609_05707_amd", "csrc")
    for f in T.KERNEL_SOURCES:
        shutil.copy(os.path.join(src, f), tmp_path / f)
    h0 = T.kernel_source_hash(str(tmp_path))
    assert h0 == T.kernel_source_hash(src)
    k = tmp_path / "decode_step.hip"
    text = k.read_text()
    k.write_text("// a new comment line\n/* and a block\n   comment */\n" + text.replace("\n", "  \n\n", 3) +
                 "\n// trailing\n")
    assert T.kernel_source_hash(str(tmp_path)) == h0
    k.write_text(text.replace("constexpr int kMergeBatch = 8;", "constexpr int kMergeBatch = 4;"))
    assert "constexpr int kMergeBatch = 8;" in text
    assert T.kernel_source_hash(str(tmp_path)) != h0
    # a "//" inside a string literal is code, not a comment
    assert T.code_only('asm("a // b");  // note') == 'asm("a // b");'
    assert T.code_only("x = '/'; /* c */ y = 1;") == "x = '/'; y = 1;"
