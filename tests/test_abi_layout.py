"""The ctypes mirrors of the executor's structs match the C layout of include/emb.h
(compiled with gcc; no GPU needed)."""
import ctypes
import os
import subprocess

import paper_2110_09132_amd as emb

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def c_layout(tmp_path, struct, fields):
    src = tmp_path / "layout.c"
    lines = ["#include <stdio.h>", "#include <stddef.h>", '#include "emb.h"', "int main(void) {",
             f'  printf("%zu\\n", sizeof({struct}));']
    lines += [f'  printf("%zu\\n", offsetof({struct}, {f}));' for f in fields]
    lines += ["  return 0;", "}"]
    src.write_text("\n".join(lines))
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-I", os.path.join(ROOT, "include"), str(src), "-o", str(exe)], check=True)
    out = subprocess.run([str(exe)], check=True, capture_output=True, text=True).stdout.split()
    return int(out[0]), [int(x) for x in out[1:]]


def test_step_args_layout(tmp_path):
    names = [f[0] for f in emb.StepArgs._fields_]
    size, offs = c_layout(tmp_path, "emb_step_args", names)
    assert size == ctypes.sizeof(emb.StepArgs)
    assert offs == [getattr(emb.StepArgs, n).offset for n in names]


def test_step_schedule_layout(tmp_path):
    names = [f[0] for f in emb.StepSchedule._fields_]
    size, offs = c_layout(tmp_path, "emb_step_schedule", names)
    assert size == ctypes.sizeof(emb.StepSchedule)
    assert offs == [getattr(emb.StepSchedule, n).offset for n in names]
