"""CPU: the host code of the C ABI (argument checks, launch planning,
workspace sizes) under AddressSanitizer and UndefinedBehaviorSanitizer.

ippd_api.hip is compiled with the sanitizers on its host side only (each
-fsanitize= behind -Xarch_host; the device code is untouched), linked with the
library's other objects into a separate libippd_san.so, and driven by a C
program built with the same sanitizers.  The program walks every entry point
through the paths that return before anything is launched (bad sizes, NULL
and misaligned pointers, missing workspaces, the no-allocation limit) and
queries workspace sizes over a sweep of shapes up to the documented maxima,
where the planner's 64-bit size arithmetic is exercised.  Any sanitizer
report fails the run (halt_on_error, no recovery)."""
import os
import shutil
import subprocess

import pytest

from paper_2609_05707_amd import build as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CLANG = "/opt/rocm/llvm/bin/clang"

C_SOURCE = r"""
#include <stddef.h>
#include <stdint.h>
#include <stdio.h>
#include <string.h>
#include "ippd.h"

#define FAKE ((void *)(size_t)0x10000)
#define MIS ((void *)(size_t)0x10009)

static void fill(ippd_batch_t *bt, int B, int nt, int hq, int hkv, int d, int dtype, int64_t pool, int maxq) {
  memset(bt, 0, sizeof *bt);
  bt->num_prompts = B; bt->num_questions = nt; bt->num_q_heads = hq; bt->num_kv_heads = hkv;
  bt->head_dim = d; bt->dtype = dtype;
  bt->ctx_pool_tokens = pool; bt->seg_capacity = 256; bt->max_ctx_len = (int32_t)(pool < 1000000 ? pool : 1000000);
  bt->max_questions = maxq; bt->rope_base = 10000.0;
  bt->ctx_off = FAKE; bt->ctx_len = FAKE; bt->q_start = FAKE; bt->seg_len = FAKE;
  bt->active = FAKE; bt->err_flag = FAKE;
}

int main(void) {
  ippd_kv_cache_t kv = {FAKE, FAKE, FAKE, FAKE};
  ippd_kv_cache_t kvmis = {MIS, FAKE, FAKE, FAKE};
  ippd_batch_t bt;
  size_t total = 0;
  int bad = 0;
  /* workspace sizes over a sweep of shapes (both dtypes and head sizes, up to
     1024 questions per prompt, 16 query heads per kv head, long pools) */
  const int dims[2] = {64, 128};
  const int groups[4] = {1, 4, 8, 16};
  const int64_t pools[4] = {8, 4096, 262144, (int64_t)1 << 24};
  const int maxqs[4] = {1, 32, 300, 1024};
  for (int dt = 0; dt < 2; ++dt)
    for (int di = 0; di < 2; ++di)
      for (int gi = 0; gi < 4; ++gi)
        for (int pi = 0; pi < 4; ++pi)
          for (int qi = 0; qi < 4; ++qi)
            for (int rows = 0; rows <= 256; rows = rows ? rows * 2 : 16) {
              const int hkv = 8, hq = hkv * groups[gi];
              fill(&bt, 64, 64 * maxqs[qi] > 200000 ? 200000 : 64 * maxqs[qi], hq, hkv, dims[di], dt, pools[pi], maxqs[qi]);
              bt.tile_rows = rows;
              for (int chunk = 0; chunk <= 4096; chunk = chunk ? chunk * 4 : 32) {
                bt.chunk_tokens = chunk;
                total += ippd_decode_workspace_bytes(&bt) + standard_decode_workspace_bytes(&bt) +
                         dense_decode_workspace_bytes(&bt);
                bt.num_instr = 3; bt.max_instr_len = 1000; bt.max_instr_questions = maxqs[qi];
                bt.instr_start = FAKE; bt.instr_off = FAKE; bt.instr_len = FAKE;
                total += ippd_decode_workspace_bytes(&bt);
                bt.num_instr = 0;
              }
            }
  /* host-side rejections of every entry point (nothing is launched) */
  fill(&bt, 2, 8, 32, 8, 128, IPPD_DTYPE_BF16, 8192, 4);
  const size_t ws = ippd_decode_workspace_bytes(&bt);
  if (ws == 0) bad |= 1;
  if (ippd_decode_attention(&bt, FAKE, &kv, FAKE, NULL, FAKE, ws - 1, NULL) != IPPD_ERR_WORKSPACE) bad |= 2;
  if (ippd_decode_attention(&bt, FAKE, &kv, NULL, NULL, FAKE, ws, NULL) != IPPD_ERR_NULL) bad |= 4;
  if (ippd_decode_attention(&bt, FAKE, &kvmis, FAKE, NULL, FAKE, ws, NULL) != IPPD_ERR_ALIGN) bad |= 8;
  if (standard_decode_attention(&bt, NULL, &kv, FAKE, NULL, FAKE, ws, NULL) != IPPD_ERR_NULL) bad |= 16;
  if (dense_decode_attention(&bt, FAKE, NULL, FAKE, NULL, FAKE, ws, NULL) != IPPD_ERR_NULL) bad |= 32;
  if (ippd_decode_step(&bt, NULL, FAKE, FAKE, NULL, &kv, FAKE, NULL, FAKE, ws, NULL) != IPPD_ERR_NULL) bad |= 64;
  if (standard_decode_step(&bt, FAKE, FAKE, MIS, NULL, &kv, FAKE, NULL, FAKE, ws, NULL) != IPPD_ERR_ALIGN) bad |= 128;
  if (ippd_append_kv(&bt, FAKE, FAKE, FAKE, NULL, &kv, NULL) != IPPD_ERR_NULL) bad |= 256;
  if (ippd_load_context(&bt, NULL, FAKE, &kv, NULL) != IPPD_ERR_NULL) bad |= 512;
  if (ippd_load_segments(&bt, FAKE, FAKE, NULL, &kv, NULL) != IPPD_ERR_NULL) bad |= 1024;
  if (ippd_load_instructions(&bt, FAKE, FAKE, &kv, NULL) != IPPD_ERR_SHAPE) bad |= 2048;
  if (ippd_prefill_attention(&bt, 8, FAKE, NULL, &kv, FAKE, FAKE, NULL) != IPPD_ERR_NULL) bad |= 4096;
  if (standard_prefill_attention(&bt, -1, FAKE, FAKE, &kv, FAKE, FAKE, NULL) != IPPD_ERR_SHAPE) bad |= 8192;
  fill(&bt, 1, 1024, 32, 8, 128, IPPD_DTYPE_BF16, 65536, 1024);
  bt.chunk_tokens = 4096;
  if (ippd_decode_step_noalloc(&bt, FAKE, FAKE, FAKE, NULL, &kv, FAKE, NULL, NULL) != IPPD_ERR_SCRATCH) bad |= 16384;
  bt.head_dim = 100;
  if (ippd_decode_step_noalloc(&bt, FAKE, FAKE, FAKE, NULL, &kv, FAKE, NULL, NULL) != IPPD_ERR_SHAPE) bad |= 32768;
  if (ippd_decode_workspace_bytes(NULL) != 0) bad |= 65536;
  if (ippd_decode_attention(NULL, FAKE, &kv, FAKE, NULL, FAKE, ws, NULL) != IPPD_ERR_NULL) bad |= 131072;
  for (int s = -1; s <= 9; ++s) total += strlen(ippd_status_string((ippd_status_t)s));
  printf("total %zu bad %d\n", total, bad);
  return bad != 0;
}
"""


def _sanitizer_runtime_dir():
    for root, _, files in os.walk("/opt/rocm/llvm/lib/clang"):
        if "libclang_rt.asan-x86_64.so" in files:
            return root
    return None


@pytest.mark.skipif(not os.path.exists(CLANG) or shutil.which(B.hipcc()) is None and not os.path.exists(B.hipcc()),
                    reason="ROCm clang / hipcc not available")
def test_host_code_under_asan_and_ubsan(tmp_path):
    rt = _sanitizer_runtime_dir()
    if rt is None:
        pytest.skip("clang sanitizer runtime not found")
    others = [os.path.join(B.BUILD_DIR, os.path.splitext(s)[0] + ".o") for s in B.SOURCES if s != "ippd_api.hip"]
    if not all(os.path.exists(o) for o in others):
        pytest.skip("library objects not built (run __graft_entry__.build())")
    san = ["-Xarch_host", "-fsanitize=address", "-Xarch_host", "-fsanitize=undefined",
           "-Xarch_host", "-fno-sanitize-recover=all", "-Xarch_host", "-fno-omit-frame-pointer"]
    api_o = tmp_path / "ippd_api_san.o"
    cmd = [B.hipcc(), *B.flags_for("ippd_api.hip"), *san, "-c", os.path.join(B.CSRC, "ippd_api.hip"),
           "-o", str(api_o)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-3000:]
    lib = tmp_path / "libippd_san.so"
    cmd = [B.hipcc(), f"--offload-arch={B.ARCH}", "-shared", "-fPIC", "-shared-libasan", *san, str(api_o), *others,
           "-o", str(lib)]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-3000:]
    src = tmp_path / "drive.c"
    src.write_text(C_SOURCE)
    exe = tmp_path / "drive"
    cmd = [CLANG, "-std=c11", "-Wall", "-Wextra", "-Werror", "-g", "-fsanitize=address,undefined",
           "-fno-sanitize-recover=all", "-shared-libasan", "-D__HIP_PLATFORM_AMD__",
           f"-I{os.path.join(ROOT, 'include')}", "-isystem", "/opt/rocm/include", str(src), "-o", str(exe),
           str(lib), f"-Wl,-rpath,{tmp_path}", f"-Wl,-rpath,{rt}", "-L/opt/rocm/lib", "-lamdhip64",
           "-Wl,-rpath,/opt/rocm/lib"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-3000:]
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=0:halt_on_error=1:abort_on_error=0",
               UBSAN_OPTIONS="halt_on_error=1:print_stacktrace=1")
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=300, env=env)
    assert "ERROR: AddressSanitizer" not in r.stderr and "runtime error" not in r.stderr, r.stderr[-3000:]
    assert r.returncode == 0, (r.stdout, r.stderr[-3000:])
    assert "bad 0" in r.stdout
