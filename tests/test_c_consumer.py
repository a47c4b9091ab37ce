"""The boundary from C: a plain C99 program includes include/decode_attn.h,
links libdecode_attn.so and calls the host-only entry points (planning,
workspace sizing, partition, error text), with no Python or torch in the
process.  The results must match the Python binding's."""

import os
import shutil
import subprocess

import pytest

import paper_2604_00028_amd as da

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
LIBDIR = os.path.join(ROOT, "paper_2604_00028_amd")

PROGRAM = r"""
#include <stdio.h>
#include "decode_attn.h"

int main(void) {
  da_plan p;
  int rc = da_choose_splits(1, 64, 8, 2048, 128, 256, 0, DA_POLICY_MI355X, &p);
  printf("choose %d %d %d %d %d %d %d %d\n", rc, p.num_splits, p.pack_gqa, p.heads_per_tile, p.tiles, p.grid,
         p.v_slices, p.combine);
  rc = da_make_plan(32, 64, 8, 8192, 128, 4, 1, 256, 0, DA_POLICY_MI355X, &p);
  printf("make %d %d %d %d\n", rc, p.num_splits, p.grid, p.combine);
  printf("workspace %zu %zu\n", da_workspace_bytes(32, 64, 128, 1), da_workspace_bytes(32, 64, 128, 4));
  int cuts[9];
  rc = da_split_bounds(5, 8, cuts);
  printf("bounds %d", rc);
  for (int i = 0; i < 9; ++i) printf(" %d", cuts[i]);
  printf("\n");
  rc = da_make_plan(0, 64, 8, 512, 128, 0, -1, 256, 0, DA_POLICY_MI355X, &p);
  printf("error %d %s\n", rc, da_strerror(rc));
  return 0;
}
"""


@pytest.mark.skipif(shutil.which("gcc") is None, reason="no C compiler")
def test_c_program_uses_the_boundary(tmp_path):
    src = tmp_path / "consumer.c"
    exe = tmp_path / "consumer"
    src.write_text(PROGRAM)
    subprocess.run(["gcc", "-std=c99", "-Wall", "-Werror", "-I", os.path.join(ROOT, "include"), str(src),
                    "-L", LIBDIR, "-ldecode_attn", f"-Wl,-rpath,{LIBDIR}", "-o", str(exe)], check=True,
                   capture_output=True)
    out = subprocess.run([str(exe)], check=True, capture_output=True, text=True, timeout=60).stdout.splitlines()
    fields = {line.split()[0]: line.split()[1:] for line in out}
    plan = da.da_choose_splits(1, 64, 8, 2048, num_cus=256)
    assert [int(x) for x in fields["choose"]] == [0, plan.num_splits, plan.pack_gqa, plan.heads_per_tile,
                                                  plan.tiles, plan.grid, plan.v_slices, plan.combine]
    forced = da.da_make_plan(32, 64, 8, 8192, num_splits=4, pack_gqa=1, num_cus=256)
    assert [int(x) for x in fields["make"]] == [0, 4, forced.grid, forced.combine]
    assert [int(x) for x in fields["workspace"]] == [0, da.da_workspace_bytes(32, 64, 128, 4)]
    assert [int(x) for x in fields["bounds"]] == [0, 0, 0, 1, 1, 2, 3, 3, 4, 5]
    assert int(fields["error"][0]) == -2 and len(" ".join(fields["error"][1:])) > 0
