"""The C-ABI library loads on the CPU and exports every function that
include/herschel.h declares (no compute calls: there may be no GPU)."""
from __future__ import annotations

import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "herschel.h")


def declared_functions():
    txt = open(HEADER).read()
    txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
    return sorted(set(re.findall(r"\b(herschel_[a-z_]+)\s*\(", txt)))


@pytest.fixture(scope="module")
def libs():
    from paper_2609_40247_amd import build, herschel
    out = []
    for variant, checked in (("release", False), ("checked", True)):
        path = herschel.library_path(variant)
        if not os.path.exists(path):
            build.build(checked=checked)
        out.append(ctypes.CDLL(path))
    return out


def test_header_declares_the_boundary():
    names = declared_functions()
    for f in ("herschel_trace_analyze", "herschel_trace_analyze_batch", "herschel_workspace_size",
              "herschel_strerror", "herschel_time_stage", "herschel_sort_stats"):
        assert f in names


def test_every_declared_symbol_is_exported(libs):
    for lib in libs:
        for f in declared_functions():
            assert hasattr(lib, f), f


def test_host_only_entry_points(libs):
    """Entry points that touch no device: sizes and messages."""
    from paper_2609_40247_amd import herschel as H
    lib = libs[0]
    lib.herschel_strerror.restype = ctypes.c_char_p
    assert lib.herschel_strerror(0) == b"ok"
    assert b"workspace" in lib.herschel_strerror(-4)
    p = H.HerschelParams(window_begin=0, window_end=30 * 10**9, gap_threshold=0, n_procs=1, n_streams=4,
                         n_threads=1, n_names=2000, n_op_names=100, flags=3)
    size = H.herschel_workspace_size(3_000_000, p, lib=H.load("release"))
    assert size > 3_000_000 * 24
    small = H.herschel_workspace_size(1000, p, lib=H.load("release"))
    assert 0 < small < size
    p.n_streams = 65
    with pytest.raises(ValueError):
        H.herschel_workspace_size(1000, p, lib=H.load("release"))
    lib.herschel_time_stage.restype = ctypes.c_int
    assert lib.herschel_time_stage(99, None, None) == -1
    assert lib.herschel_time_stage(1, None, None) == 0
    lib.herschel_sort_stats.restype = ctypes.c_int
    assert lib.herschel_sort_stats(None, None) == -1


def test_struct_layouts_match_the_header(tmp_path):
    """The binding's ctypes structures (and the edge record's numpy dtype)
    have the header's sizes and field offsets, as the host C compiler lays
    them out."""
    from paper_2609_40247_amd import herschel as H
    from paper_2609_40247_amd import synth
    structs = {"herschel_events": H.HerschelEvents, "herschel_params": H.HerschelParams,
               "herschel_outputs": H.HerschelOutputs}
    lines = ['#include <stddef.h>', '#include <stdio.h>', '#include "herschel.h"', "int main(void) {"]
    for cname, cls in structs.items():
        lines.append(f'  printf("{cname} %zu\\n", sizeof({cname}));')
        for f, _ in cls._fields_:
            lines.append(f'  printf("{cname}.{f} %zu\\n", offsetof({cname}, {f}));')
    lines.append('  printf("herschel_edge %zu\\n", sizeof(herschel_edge));')
    for f in synth.EDGE_DTYPE.names:
        lines.append(f'  printf("herschel_edge.{f} %zu\\n", offsetof(herschel_edge, {f}));')
    lines.append('  printf("herschel_counters %zu\\n", sizeof(herschel_counters));')
    lines += ["  return 0;", "}"]
    src = tmp_path / "layout.c"
    src.write_text("\n".join(lines) + "\n")
    exe = tmp_path / "layout"
    import subprocess
    subprocess.run(["gcc", "-std=c11", "-I", os.path.join(ROOT, "include"), "-o", str(exe), str(src)], check=True)
    got = dict(line.rsplit(" ", 1) for line in subprocess.run([str(exe)], check=True, capture_output=True,
                                                                 text=True).stdout.splitlines())
    for cname, cls in structs.items():
        assert int(got[cname]) == ctypes.sizeof(cls), cname
        for f, _ in cls._fields_:
            assert int(got[f"{cname}.{f}"]) == getattr(cls, f).offset, f"{cname}.{f}"
    assert int(got["herschel_edge"]) == synth.EDGE_DTYPE.itemsize
    for f in synth.EDGE_DTYPE.names:
        assert int(got[f"herschel_edge.{f}"]) == synth.EDGE_DTYPE.fields[f][1], f
    assert int(got["herschel_counters"]) == 8 * len(H.COUNTERS)


def test_oracle_struct_layouts(tmp_path):
    """The oracle wrapper's ctypes structures match the oracle's header."""
    import subprocess

    import oracle
    structs = {"hro_events": oracle._Events, "hro_params": oracle._Params, "hro_outputs": oracle._Outputs}
    lines = ['#include <stddef.h>', '#include <stdio.h>', '#include "herschel_oracle.h"', "int main(void) {"]
    for cname, cls in structs.items():
        lines.append(f'  printf("{cname} %zu\\n", sizeof({cname}));')
        for f, _ in cls._fields_:
            lines.append(f'  printf("{cname}.{f} %zu\\n", offsetof({cname}, {f}));')
    lines += ["  return 0;", "}"]
    src = tmp_path / "layout.c"
    src.write_text("\n".join(lines) + "\n")
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-std=c11", "-I", os.path.join(ROOT, "oracle"), "-o", str(exe), str(src)], check=True)
    got = dict(line.rsplit(" ", 1) for line in subprocess.run([str(exe)], check=True, capture_output=True,
                                                                 text=True).stdout.splitlines())
    for cname, cls in structs.items():
        assert int(got[cname]) == ctypes.sizeof(cls), cname
        for f, _ in cls._fields_:
            assert int(got[f"{cname}.{f}"]) == getattr(cls, f).offset, f"{cname}.{f}"
