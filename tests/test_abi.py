"""The C-ABI library: it loads, exports every function include/mas.h declares,
and rejects invalid arguments on the host before touching the GPU."""
from __future__ import annotations

import ctypes
import os
import re
import subprocess

import pytest

import paper_2409_07704_amd as mas
from paper_2409_07704_amd import _native

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "mas.h")


def declared_functions():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(mas_[a-z_]+)\s*\(", src)))


def test_header_declares_the_boundary():
    assert declared_functions() == sorted(_native.SIGNATURES)


def test_library_exports_every_declared_symbol():
    lib = mas.lib()
    for name in declared_functions():
        assert hasattr(lib, name), name
    out = subprocess.run(["nm", "-D", "--defined-only", mas.LIB_PATH], capture_output=True, text=True).stdout
    exported = set(re.findall(r" T (mas_\w+)", out))
    assert set(declared_functions()) <= exported


def test_version_and_status_strings():
    assert mas.mas_version() == 2
    assert mas.mas_status_string(0) == "MAS_OK"
    assert mas.mas_status_string(3) == "MAS_ERR_WORKSPACE"
    assert mas.mas_status_string(99) == "MAS_ERR_UNKNOWN"


def test_workspace_bytes():
    assert mas.mas_workspace_bytes(0, 10, 10) == 0
    assert mas.mas_workspace_bytes(1, 0, 10) == 0
    assert mas.mas_workspace_bytes(1, 10, -1) == 0
    n = mas.mas_workspace_bytes(64, 1024, 4096)
    assert n % 256 == 0
    # decision words: 1 bit per cell rounded to 32-column words of 64-row waves
    assert n >= 64 * 128 * 1024 * 4
    assert mas.mas_workspace_bytes(64, 1024, 4097) > n
    # sizes whose product overflows are refused
    assert mas.mas_workspace_bytes(2**30, 2**20, 2**20) == 0
    # T above the on-chip row_start table, and item slabs of 2 GiB or more
    assert mas.mas_workspace_bytes(1, 8192, 16) > 0
    assert mas.mas_workspace_bytes(1, 8193, 16) == 0
    assert mas.mas_workspace_bytes(1, 8192, 65535) > 0
    assert mas.mas_workspace_bytes(1, 8192, 65536) == 0


FAKE = ctypes.c_void_p(0x10000)  # never dereferenced: validation fails first


@pytest.mark.parametrize(
    "args,code",
    [
        # value, t_x, t_y, B, T, S, row_start, durations, score, status, workspace, bytes, stream
        ((None, FAKE, FAKE, 1, 1, 1, FAKE, None, None, None, FAKE, 1 << 20, None), 1),
        ((FAKE, None, FAKE, 1, 1, 1, FAKE, None, None, None, FAKE, 1 << 20, None), 1),
        ((FAKE, FAKE, FAKE, 1, 1, 1, None, None, None, None, FAKE, 1 << 20, None), 1),
        ((FAKE, FAKE, FAKE, 0, 1, 1, FAKE, None, None, None, FAKE, 1 << 20, None), 2),
        ((FAKE, FAKE, FAKE, 1, -5, 1, FAKE, None, None, None, FAKE, 1 << 20, None), 2),
        ((FAKE, FAKE, FAKE, 1, 1, 1, FAKE, None, None, None, None, 1 << 20, None), 3),
        ((FAKE, FAKE, FAKE, 1, 1, 1, FAKE, None, None, None, ctypes.c_void_p(0x10010), 1 << 20, None), 3),
        ((FAKE, FAKE, FAKE, 4, 64, 64, FAKE, None, None, None, FAKE, 256, None), 3),
    ],
)
def test_mas_search_host_validation(args, code):
    assert mas.lib().mas_search(*args) == code


def test_other_entry_points_host_validation():
    L = mas.lib()
    assert L.mas_forward_ex(None, FAKE, FAKE, FAKE, 1, 1, 1, None, None, FAKE, 1 << 20, None) == 1
    assert L.mas_forward_ex(FAKE, FAKE, FAKE, FAKE, 1, 1, 0, None, None, FAKE, 1 << 20, None) == 2
    assert L.mas_forward_ex(FAKE, FAKE, FAKE, FAKE, 8, 8, 8, None, None, FAKE, 16, None) == 3
    assert L.mas_forward(FAKE, FAKE, None, FAKE, 1, 1, 1, None) == 1
    assert L.mas_forward(FAKE, FAKE, FAKE, FAKE, 1, 0, 1, None) == 2
    assert L.mas_expand_path(None, 1, 1, 1, FAKE, None) == 1
    assert L.mas_expand_path(FAKE, -1, 1, 1, FAKE, None) == 2
    # the text grid: pointers, shape limits and element widths
    assert L.mas_expand_text(None, FAKE, 1, 1, 1, 1, 4, FAKE, None) == 1
    assert L.mas_expand_text(FAKE, None, 1, 1, 1, 1, 4, FAKE, None) == 1
    assert L.mas_expand_text(FAKE, FAKE, 1, 1, 1, 1, 4, None, None) == 1
    for bad in ((0, 1, 1, 1, 4), (1, 0, 1, 1, 4), (1, 1, 0, 1, 4), (1, 1, 1, 0, 4), (1, 1, 1, 1, 3), (1, 1, 1, 1, 16),
                (1, 1, 1, 1 << 22, 8), (1 << 20, 8, 1 << 20, 1 << 10, 4)):
        assert L.mas_expand_text(FAKE, FAKE, *bad[:4], bad[4], FAKE, None) == 2, bad
    assert L.mas_workspace_init(None, 256, None) == 1
    assert L.mas_workspace_init(ctypes.c_void_p(0x10008), 256, None) == 3
    assert L.mas_workspace_init(FAKE, 100, None) == 3
    # the log-likelihood producer
    assert L.mas_loglik(None, None, FAKE, FAKE, FAKE, 1, 1, 1, 8, FAKE, None) == 1
    assert L.mas_loglik(FAKE, None, FAKE, FAKE, FAKE, 1, 1, 1, 8, None, None) == 1
    assert L.mas_loglik(FAKE, None, FAKE, FAKE, FAKE, 1, 1, 1, 0, FAKE, None) == 2
    assert L.mas_loglik(FAKE, None, FAKE, FAKE, FAKE, 1, 1, 1, 193, FAKE, None) == 2
    assert L.mas_loglik(FAKE, None, FAKE, FAKE, FAKE, 1, 8193, 1, 8, FAKE, None) == 2
    # the static-scratch entry point: checked before any device call
    assert L.mas_forward_static(None, FAKE, FAKE, FAKE, 1, 1, 1, None, None, None) == 1
    assert L.mas_forward_static(FAKE, FAKE, FAKE, FAKE, 1, 0, 1, None, None, None) == 2
    assert mas.mas_workspace_bytes(64, 1024, 8192) > mas.STATIC_SCRATCH_BYTES
    assert L.mas_forward_static(FAKE, FAKE, FAKE, FAKE, 64, 1024, 8192, None, None, None) == 5
    assert mas.mas_status_string(5) == "MAS_ERR_SCRATCH"
    # the legacy-sentinel mode: a finite negative sentinel only
    for bad in (float("nan"), float("inf"), float("-inf"), 0.0, 1e9):
        assert L.mas_forward_sentinel(FAKE, FAKE, FAKE, FAKE, 1, 1, 1, bad, None, None, FAKE, 1 << 20, None) == 6
    assert L.mas_forward_sentinel(FAKE, FAKE, FAKE, FAKE, 1, 0, 1, -1e9, None, None, FAKE, 1 << 20, None) == 2
    assert L.mas_forward_sentinel(FAKE, None, FAKE, FAKE, 1, 1, 1, -1e9, None, None, FAKE, 1 << 20, None) == 1
    assert mas.mas_status_string(6) == "MAS_ERR_BAD_VALUE"


def test_binding_refuses_host_tensors():
    import torch

    v = torch.zeros(1, 2, 3)
    x = torch.ones(1, dtype=torch.int32)
    with pytest.raises(TypeError):
        mas.mas_forward(v, x, x)
