"""CPU: the boundary as C sees it.  A C11 program compiled by gcc against
include/ippd.h (-Wall -Wextra -Werror) and linked to libippd.so calls the
entry points that validate and plan without launching anything.  Its struct
sizes and field offsets must equal the ctypes mirror's, and its results the
ones the binding gets for the same batch."""
import ctypes
import os
import shutil
import subprocess

import pytest

from paper_2609_05707_amd import _lib as L

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PKG = os.path.join(ROOT, "paper_2609_05707_amd")

FIELDS = [f for f, _ in L.IppdBatch._fields_]

C_SOURCE = r"""
#include <stddef.h>
#include <stdio.h>
#include <string.h>
#include "ippd.h"

static void fill(ippd_batch_t *bt) {
  memset(bt, 0, sizeof *bt);
  bt->num_prompts = 1; bt->num_questions = 4; bt->num_q_heads = 4; bt->num_kv_heads = 2;
  bt->head_dim = 64; bt->dtype = IPPD_DTYPE_F32;
  bt->ctx_pool_tokens = 256; bt->seg_capacity = 32; bt->max_ctx_len = 256; bt->max_questions = 4;
  bt->rope_base = 10000.0;
  void *fake = (void *)(size_t)0x10000;
  bt->ctx_off = fake; bt->ctx_len = fake; bt->q_start = fake; bt->seg_len = fake;
  bt->active = fake; bt->err_flag = fake;
}

int main(void) {
  printf("size batch %zu\n", sizeof(ippd_batch_t));
  printf("size kv %zu\n", sizeof(ippd_kv_cache_t));
%OFFSETS%
  printf("version %d\n", ippd_version());
  for (int s = 0; s <= 6; ++s) printf("status %d %s\n", s, ippd_status_string((ippd_status_t)s));
  ippd_batch_t bt;
  fill(&bt);
  printf("workspace %zu\n", ippd_decode_workspace_bytes(&bt));
  printf("standard_workspace %zu\n", standard_decode_workspace_bytes(&bt));
  printf("load_null %d\n", (int)ippd_load_context(&bt, NULL, NULL, NULL, NULL));
  bt.head_dim = 96;
  printf("bad_head_dim %d\n", (int)ippd_load_context(&bt, (void *)1, (void *)1, NULL, NULL));
  return 0;
}
"""


def _valid_batch():
    bt = L.IppdBatch()
    bt.num_prompts, bt.num_questions, bt.num_q_heads, bt.num_kv_heads = 1, 4, 4, 2
    bt.head_dim, bt.dtype = 64, L.IPPD_DTYPE_F32
    bt.ctx_pool_tokens, bt.seg_capacity, bt.max_ctx_len, bt.max_questions = 256, 32, 256, 4
    bt.rope_base = 10000.0
    for f in ("ctx_off", "ctx_len", "q_start", "seg_len", "active", "err_flag"):
        setattr(bt, f, 0x10000)
    return bt


@pytest.fixture(scope="module")
def c_run(tmp_path_factory):
    gcc = shutil.which("gcc")
    if gcc is None:
        pytest.skip("gcc not available")
    if not os.path.exists(os.path.join(PKG, "libippd.so")):
        pytest.fail("libippd.so is not built")
    d = tmp_path_factory.mktemp("c_abi")
    offsets = "\n".join(f'  printf("off {f} %zu\\n", offsetof(ippd_batch_t, {f}));' for f in FIELDS)
    src = d / "abi.c"
    src.write_text(C_SOURCE.replace("%OFFSETS%", offsets))
    exe = d / "abi"
    cmd = [gcc, "-std=c11", "-Wall", "-Wextra", "-Werror", "-D__HIP_PLATFORM_AMD__",
           f"-I{os.path.join(ROOT, 'include')}", "-isystem", "/opt/rocm/include", str(src), "-o", str(exe),
           f"-L{PKG}", "-l:libippd.so", f"-Wl,-rpath,{PKG}"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stderr
    out = {}
    for line in r.stdout.splitlines():
        k, rest = line.split(" ", 1)
        out.setdefault(k, []).append(rest)
    return out


def test_layout_matches_the_binding(c_run):
    assert int(c_run["size"][0].split()[1]) == ctypes.sizeof(L.IppdBatch)
    assert int(c_run["size"][1].split()[1]) == ctypes.sizeof(L.IppdKvCache)
    offs = dict(x.split() for x in c_run["off"])
    for f in FIELDS:
        assert int(offs[f]) == getattr(L.IppdBatch, f).offset, f


def test_results_match_the_binding(c_run):
    lib = L.load_library()
    assert int(c_run["version"][0]) == lib.ippd_version()
    for line in c_run["status"]:
        s, text = line.split(" ", 1)
        assert text == lib.ippd_status_string(int(s)).decode()
    bt = _valid_batch()
    assert int(c_run["workspace"][0]) == lib.ippd_decode_workspace_bytes(ctypes.byref(bt)) > 0
    assert int(c_run["standard_workspace"][0]) == lib.standard_decode_workspace_bytes(ctypes.byref(bt)) > 0
    assert int(c_run["load_null"][0]) == L.IPPD_ERR_NULL
    assert int(c_run["bad_head_dim"][0]) == L.IPPD_ERR_SHAPE
