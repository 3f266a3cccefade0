"""The C ABI on a machine without a GPU: the library loads, exports exactly
what include/sifar.h declares, and rejects bad configurations on the host
before any device call."""
from __future__ import annotations

import ctypes
import os
import re

import pytest

import paper_2607_08973_amd as S

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include",
                      "sifar.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(sifar_[a-z_]+)\s*\(", text)))


def test_header_declares_the_binding_exports():
    assert declared_functions() == sorted(S.EXPORTS)


def test_library_exports_every_declared_symbol():
    lib = S.load()
    for name in declared_functions():
        assert hasattr(lib, name), name


def test_struct_layouts_match_header():
    # sifar_config: 16 four-byte fields; sifar_step_buffers: pointer/int64 layout
    assert ctypes.sizeof(S.sifar_config) == 64
    assert ctypes.sizeof(S.sifar_step_buffers) == 64
    text = open(HEADER).read()
    cfg = re.search(r"typedef struct \{([^{}]*)\} sifar_config;", text).group(1)
    fields = re.findall(r"\b(?:int32_t|uint32_t|float)\s+(\w+);", cfg)
    assert fields == [f for f, _ in S.sifar_config._fields_]
    buf = re.search(r"typedef struct \{([^{}]*)\} sifar_step_buffers;", text).group(1)
    bfields = re.findall(r"\b(\w+);", buf)
    assert bfields == [f for f, _ in S.sifar_step_buffers._fields_]


def test_defaults_and_strings():
    c = S.sifar_config_default()
    assert (c.nranks, c.hidden, c.max_tokens, c.reduces_per_step) == (8, 4096, 8, 64)
    assert c.validate == S.SIFAR_VALIDATE_SPEC and c.epilogue == 0
    assert abs(c.rms_eps - 1e-6) < 1e-12
    assert c.max_attempts == 1 << 20 and c.waves_per_group == 1 and c.fuse_peers == 1
    assert c.persistent == 0 and c.late_delay == 8 and c.buffers == 2
    assert S.sifar_version() >= 100
    for code in (0, -1, -2, -3, -4, -5):
        assert S.strerror(code)
    assert S.strerror(-99) == "unknown error"


@pytest.mark.parametrize("field,value", [
    ("nranks", 0), ("nranks", 9), ("hidden", 4), ("hidden", 4100), ("hidden", 65544),
    ("max_tokens", 0), ("reduces_per_step", 0), ("validate", 3), ("epilogue", 2),
    ("max_attempts", 0), ("spin_limit", 0), ("log_epochs", 0), ("waves_per_group", 3),
    ("waves_per_group", 32), ("fuse_peers", 2), ("persistent", 2), ("buffers", 0), ("buffers", 3),
])
def test_invalid_config_rejected_on_host(field, value):
    c = S.sifar_config_default()
    setattr(c, field, value)
    h = ctypes.c_void_p()
    rc = S.load().sifar_init(ctypes.byref(c), ctypes.byref(h))
    assert rc == S.SIFAR_EINVAL and not h.value


@pytest.mark.parametrize("mode", [0, 2])  # SPEC, NONE
def test_persistent_step_requires_ordered_validation(mode):
    """A persistent step reads slots its peers are writing: without validation
    the reads race the writes, and speculative loads were measured to return
    stale ranks whose stamps read fresh; only ORDERED is accepted."""
    c = S.sifar_config_default()
    c.persistent = 1
    c.validate = mode
    h = ctypes.c_void_p()
    assert S.load().sifar_init(ctypes.byref(c), ctypes.byref(h)) == S.SIFAR_EINVAL
    assert not h.value


def test_null_handle_rejected():
    L = S.load()
    assert L.sifar_reduce(None, None, 1, None) == S.SIFAR_EINVAL
    assert L.sifar_step(None, 1, None) == S.SIFAR_EINVAL
    assert L.sifar_status(None) == S.SIFAR_EINVAL
    assert L.sifar_init(None, None) == S.SIFAR_EINVAL
    L.sifar_destroy(None)


def test_floor_constants_match_header():
    text = open(HEADER).read()
    block = re.search(r"enum \{([^{}]*SIFAR_FLOOR_[^{}]*)\};", text).group(1)
    pairs = dict((k, int(v)) for k, v in re.findall(r"(SIFAR_FLOOR_\w+)\s*=\s*(\d+)", block))
    assert len(pairs) == 10
    for k, v in pairs.items():
        assert getattr(S, k) == v, k


@pytest.mark.parametrize("kind,iterations", [
    (-1, 10), (10, 10),                                   # unknown kinds
    (S.SIFAR_FLOOR_ATOMIC, 0), (S.SIFAR_FLOOR_ATOMIC, (1 << 20) + 1),
    (S.SIFAR_FLOOR_GRAPH_NODE, 4097), (S.SIFAR_FLOOR_EAGER_LAUNCH, 4097),
    (S.SIFAR_FLOOR_COLD_LOAD, 65537), (S.SIFAR_FLOOR_PINGPONG_XCD, 65537),
    (S.SIFAR_FLOOR_PINGPONG_SAME_XCD, 65537),
])
def test_floor_rejects_bad_arguments_on_host(kind, iterations):
    L = S.load()
    ns = ctypes.c_double(-1.0)
    info = (ctypes.c_uint32 * 4)()
    assert L.sifar_floor(kind, iterations, None, ctypes.byref(ns), info) == S.SIFAR_EINVAL
    assert L.sifar_floor(S.SIFAR_FLOOR_ATOMIC, 10, None, None, info) == S.SIFAR_EINVAL
    assert L.sifar_floor(S.SIFAR_FLOOR_ATOMIC, 10, None, ctypes.byref(ns), None) == S.SIFAR_EINVAL


@pytest.mark.parametrize("protocol,placement,pairs,trials", [
    (3, 0, 8, 10), (-1, 0, 8, 10), (0, 2, 8, 10), (0, 0, 0, 10), (0, 0, 12, 10),
    (0, 0, 520, 10), (0, 0, 8, 0), (0, 0, 8, (1 << 20) + 1),
])
def test_litmus_rejects_bad_arguments(protocol, placement, pairs, trials):
    L = S.load()
    r = S.sifar_litmus_result()
    assert L.sifar_litmus(protocol, placement, pairs, trials, None, ctypes.byref(r)) == S.SIFAR_EINVAL
    assert L.sifar_litmus(0, 0, 8, 10, None, None) == S.SIFAR_EINVAL


def test_every_numeric_define_matches_the_binding():
    text = open(HEADER).read()
    defs = re.findall(r"#define (SIFAR_\w+)\s+\(?(-?\d+)\)?", text)
    assert len(defs) >= 15
    for k, v in defs:
        assert getattr(S, k) == int(v), k


def test_litmus_result_layout_matches_header():
    text = open(HEADER).read()
    body = re.search(r"typedef struct \{([^{}]*)\} sifar_litmus_result;", text).group(1)
    fields = re.findall(r"\b(\w+)(?:\[\d+\])?;", body)
    assert fields == [f for f, _ in S.sifar_litmus_result._fields_]
    assert ctypes.sizeof(S.sifar_litmus_result) == 4 * 8 + 2 * 4 + 8 + 4 * 4


def test_struct_offsets_match_a_c_compiler(tmp_path):
    """The ctypes mirrors against what a C compiler makes of the header."""
    import shutil
    import subprocess

    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        pytest.skip("no C compiler")
    structs = {"sifar_config": S.sifar_config, "sifar_step_buffers": S.sifar_step_buffers,
               "sifar_litmus_result": S.sifar_litmus_result}
    lines = ["#include <stdio.h>", "#include <stddef.h>", '#include "sifar.h"', "int main(void) {"]
    for name, cls in structs.items():
        lines.append(f'    printf("{name} size %zu\\n", sizeof({name}));')
        for f, _ in cls._fields_:
            lines.append(f'    printf("{name} {f} %zu\\n", offsetof({name}, {f}));')
    lines += ["    return 0;", "}"]
    src = tmp_path / "layout.c"
    src.write_text("\n".join(lines) + "\n")
    exe = tmp_path / "layout"
    subprocess.run([cc, "-std=c11", "-I", os.path.dirname(HEADER), str(src), "-o", str(exe)],
                   check=True)
    got = subprocess.run([str(exe)], check=True, capture_output=True, text=True).stdout.split("\n")
    for line in filter(None, got):
        name, what, value = line.split()
        cls = structs[name]
        want = ctypes.sizeof(cls) if what == "size" else getattr(cls, what).offset
        assert int(value) == want, line


@pytest.mark.parametrize("nranks,tokens,hidden,stride,misalign", [
    (0, 1, 4096, 4096, 0), (9, 1, 4096, 4096, 0),          # ranks
    (2, 0, 4096, 4096, 0), (2, 65, 4096, 65 * 4096, 0),    # tokens
    (2, 1, 4100, 4100, 0), (2, 1, 0, 8, 0),                # hidden
    (2, 64, 8192, 64 * 8192, 0),                           # beyond the static array
    (2, 2, 4096, 4096, 0), (2, 1, 4096, 4100, 0),          # rank stride
    (2, 1, 4096, 4096, 8),                                 # 8-byte aligned pointers
])
def test_noalloc_rejects_out_of_range_calls_on_host(nranks, tokens, hidden, stride, misalign):
    """The allocation-free entry point refuses, before any device call, every
    size its static array cannot hold and every malformed argument."""
    L = S.load()
    buf = ctypes.create_string_buffer(64)
    p = (ctypes.addressof(buf) + 15) // 16 * 16 + misalign
    assert L.sifar_allreduce_noalloc(p, stride, nranks, tokens, hidden, p, None) == S.SIFAR_EINVAL
    assert L.sifar_allreduce_noalloc(None, 4096, 2, 1, 4096, p, None) == S.SIFAR_EINVAL
