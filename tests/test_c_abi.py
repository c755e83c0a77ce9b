"""The C ABI from C: every header compiles as strict C99 and C++11, and a C program linked
against the library gets the same host-side answers (workspace size, visible pairs, plan
size, status text, refusals) as the Python binding.  Host calls only: nothing here
touches a GPU."""
import os
import shutil
import subprocess

import pytest

from paper_2609_34318_amd import hydra

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
INC = os.path.join(ROOT, "include")
PKG = os.path.join(ROOT, "paper_2609_34318_amd")

pytestmark = pytest.mark.skipif(shutil.which("gcc") is None, reason="gcc not available")

HEADERS = sorted(h for h in os.listdir(INC) if h.endswith(".h"))

PROGRAM = r"""
#include <stdio.h>
#include <string.h>
#include "hydra_attn.h"

int main(void) {
  int32_t cu[4] = {0, 64, 192, 512};
  int32_t items[64 * 16];
  int32_t qt = 0, kt = 0;
  hydra_problem_t p;
  memset(&p, 0, sizeof p);
  p.n_heads = 4;
  p.d_qk = 192;
  p.d_v = 128;
  p.cu_seqlens = cu;
  p.n_docs = 3;
  p.q.n_segs = 1;
  p.q.len[0] = 512;
  p.kv.n_segs = 2;
  p.kv.start[0] = 0;
  p.kv.len[0] = 100;
  p.kv.start[1] = 300;
  p.kv.len[1] = 40;
  printf("ws %zu\n", hydra_workspace_size(&p));
  printf("pairs %lld\n", (long long)hydra_visible_pairs(&p));
  printf("qitems %lld\n", (long long)hydra_plan_items(&p, 0, items, 64));
  printf("kitems %lld\n", (long long)hydra_plan_items(&p, 1, items, 64));
  hydra_tile_rows(&qt, &kt);
  printf("tiles %d %d\n", qt, kt);
  printf("status %s\n", hydra_strerror(HYDRA_ERR_WORKSPACE));
  /* refusals before any HIP call */
  printf("fwd_null %d\n", hydra_attn_fwd(&p, NULL, NULL, NULL, NULL, NULL, NULL, NULL, 0, NULL));
  p.d_qk = 128;
  printf("unsupported %d\n", hydra_attn_fwd(&p, NULL, NULL, NULL, NULL, NULL, NULL, NULL, 0, NULL));
  p.d_qk = 192;
  p.q_tok_stride = 4 * 192 + 4;
  printf("bad_stride %zu\n", hydra_workspace_size(&p));
  return 0;
}
"""


@pytest.fixture(scope="module")
def lib_path():
    if not os.path.exists(hydra.LIB_PATH):
        from paper_2609_34318_amd import build_lib
        build_lib.build()
    return hydra.LIB_PATH


@pytest.mark.parametrize("lang", ["c99", "c++11"])
def test_headers_compile_strictly(tmp_path, lang):
    src = tmp_path / "all.c"
    src.write_text("".join(f'#include "{h}"\n' for h in HEADERS) + "int main(void) { return 0; }\n")
    cmd = ["gcc", f"-std={lang}", "-Wall", "-Wextra", "-pedantic", "-Werror", f"-I{INC}", "-c", str(src),
           "-o", str(tmp_path / "all.o")]
    if lang.startswith("c++"):
        cmd[0:1] = ["g++", "-x", "c++"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr


def test_c_program_matches_the_binding(tmp_path, lib_path):
    src = tmp_path / "prog.c"
    src.write_text(PROGRAM)
    exe = tmp_path / "prog"
    r = subprocess.run(["gcc", "-std=c99", "-Wall", "-Werror", f"-I{INC}", str(src), f"-L{PKG}", "-lhydra_attn",
                        f"-Wl,-rpath,{PKG}", "-Wl,-rpath-link,/opt/rocm/lib", "-o", str(exe)],
                       capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=60)
    assert r.returncode == 0, r.stderr
    got = dict(line.split(" ", 1) for line in r.stdout.strip().splitlines())
    p = hydra.Problem([0, 64, 192, 512], 4, [(0, 512)], [(0, 100), (300, 40)])
    assert int(got["ws"]) == hydra.workspace_size(p) > 0
    assert int(got["pairs"]) == hydra.visible_pairs(p)
    assert int(got["qitems"]) == len(hydra.plan_items(p, 0))
    assert int(got["kitems"]) == len(hydra.plan_items(p, 1))
    assert got["tiles"] == "%d %d" % hydra.tile_rows()
    assert got["status"] == hydra.lib().hydra_strerror(-4).decode()
    assert int(got["fwd_null"]) == -1 and int(got["unsupported"]) == -2 and int(got["bad_stride"]) == 0


@pytest.mark.gpu
def test_c_program_runs_the_forward_without_torch(tmp_path, lib_path):
    """tests/c_abi_forward.c: hipMalloc'd buffers, hydra_attn_fwd from C, the uniform-softmax
    closed form checked in the program itself."""
    exe = tmp_path / "c_abi_forward"
    r = subprocess.run(["gcc", "-std=c99", "-Wall", "-Werror", "-D__HIP_PLATFORM_AMD__", "-I/opt/rocm/include",
                        f"-I{INC}", os.path.join(ROOT, "tests", "c_abi_forward.c"), f"-L{PKG}", "-lhydra_attn",
                        "-L/opt/rocm/lib", "-lamdhip64", "-lm", f"-Wl,-rpath,{PKG}", "-Wl,-rpath,/opt/rocm/lib",
                        "-o", str(exe)], capture_output=True, text=True)
    assert r.returncode == 0, r.stderr
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=120)
    print(r.stdout.strip())
    assert r.returncode == 0, r.stdout + r.stderr
