"""CPU checks of the C ABI: the library loads, exports every symbol that
include/ssn.h declares, and rejects bad arguments on the host before any HIP
call (fake device addresses are never dereferenced on these paths)."""
import ctypes
import os
import re
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "ssn.h")

OK, ERR_NULL, ERR_SHAPE, ERR_DTYPE, ERR_ALIGN, ERR_UNSUPPORTED, ERR_LAUNCH, ERR_ALIAS = range(8)


@pytest.fixture(scope="module")
def ssn():
    from paper_2607_13332_amd import ssn as mod
    if not os.path.exists(mod.LIB_PATH):
        from paper_2607_13332_amd import build
        build.build(verbose=False)
    mod.lib()
    return mod


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(ssn_[a-z_]+)\s*\(", text)))


def test_header_declares_the_four_codec_operations():
    names = declared_functions()
    for n in ("ssn_compress", "ssn_decompress", "ssn_project_grad", "ssn_project_weights"):
        assert n in names


def test_every_declared_symbol_is_exported(ssn):
    out = subprocess.run(["nm", "-D", "--defined-only", ssn.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = set(l.split()[-1] for l in out.splitlines() if l.strip())
    missing = [n for n in declared_functions() if n not in exported]
    assert not missing, missing
    for n in declared_functions():
        assert hasattr(ssn.lib(), n)


def test_version_and_status_strings(ssn):
    L = ssn.lib()
    assert L.ssn_abi_version() == 3
    assert L.ssn_status_string(OK) == b"ok"
    assert L.ssn_status_string(ERR_ALIAS) == b"output overlaps an input"
    assert L.ssn_status_string(99) == b"unknown status"


def test_kernel_family_rules(ssn):
    kf = ssn.kernel_family
    assert kf("compress", "bf16", 4096, 64) == "mfma"
    assert kf("compress", "bf16", 4096, 128) == "mfma"
    assert kf("compress", "bf16", 4096, 129) == "generic"
    assert kf("compress", "bf16", 4100, 64) == "generic"
    assert kf("compress", "f32", 256, 8) == "mfma"
    assert kf("compress", "f32", 4000, 8) == "generic"
    assert kf("project_grad", "bf16", 2048, 32) == "mfma"
    assert kf("decompress", "bf16", 4096, 64) == "mfma"
    assert kf("decompress", "bf16", 4096, 51) == "mfma"
    assert kf("decompress", "bf16", 5120, 1) == "mfma"
    assert kf("decompress", "bf16", 4096, 129) == "generic"
    assert kf("project_weights", "bf16", 5120, 51) == "mfma"
    assert kf("decompress", "bf16", 4064, 64) == "generic"
    assert kf("project_weights", "bf16", 4096, 64) == "mfma"
    assert kf("project_weights", "f32", 4096, 64) == "mfma"
    assert kf("project_weights", "f32", 5120, 51) == "mfma"
    assert kf("project_weights", "f32", 4100, 64) == "generic"
    assert kf("project_weights", "f32", 4096, 144) == "generic"
    assert kf("compress_projected", "bf16", 4096, 64) == "mfma"
    assert kf("compress_projected", "bf16", 5120, 51) == "mfma"
    # float32 storage: the matrix-core kernels where d is a multiple of 64 and
    # U rows hold 16, 32, .., 128 floats; generic otherwise
    assert kf("compress_projected", "f32", 4096, 64) == "mfma"
    assert kf("compress", "f32", 5120, 16) == "mfma"
    assert kf("decompress", "f32", 4096, 128) == "mfma"
    assert kf("project_grad", "f32", 4096, 51) == "mfma"
    assert kf("decompress", "f32", 5120, 1) == "mfma"
    assert kf("decompress", "f32", 4096, 144) == "generic"
    assert kf("decompress", "f32", 4100, 64) == "generic"
    assert ssn.lib().ssn_kernel_family(9, 1, 4096, 64) == b"invalid"


# Fake, never-dereferenced device addresses (16-byte aligned, far apart).
A = 0x7F0000000000
B = 0x7F1000000000
C = 0x7F2000000000
D = 0x7F3000000000
F = 0x7F4000000000


def test_compress_validation(ssn):
    f = ssn.lib().ssn_compress
    assert f(7, 10, 64, 8, 100, A, B, C, D, F, None) == ERR_DTYPE
    assert f(1, -1, 64, 8, 100, A, B, C, D, F, None) == ERR_SHAPE
    assert f(1, 10, 64, 65, 100, A, B, C, D, F, None) == ERR_SHAPE      # k > d
    assert f(1, 10, 64, 0, 100, A, B, C, D, F, None) == ERR_SHAPE
    assert f(1, 10, 64, 8, 0, A, B, C, D, F, None) == ERR_SHAPE        # V < 1
    assert f(1, 1 << 40, 1 << 30, 8, 100, A, B, C, D, F, None) == ERR_SHAPE   # overflow
    assert f(1, 0, 64, 8, 100, None, None, None, None, None, None) == OK   # N == 0 no-op
    assert f(1, 10, 64, 8, 100, None, B, C, D, F, None) == ERR_NULL
    assert f(1, 10, 64, 8, 100, A, B, C, D, None, None) == ERR_NULL
    assert f(1, 10, 64, 8, 100, A + 1, B, C, D, F, None) == ERR_ALIGN   # bf16 needs 2 B
    assert f(0, 10, 64, 8, 100, A + 2, B, C, D, F, None) == ERR_ALIGN   # fp32 needs 4 B
    assert f(1, 10, 64, 8, 100, A, B + 2, C, D, F, None) == ERR_ALIGN   # ids int32
    # Z overlapping X / U / E
    assert f(1, 10, 64, 8, 100, A, B, C, D, A + 64, None) == ERR_ALIAS
    assert f(1, 10, 64, 8, 100, A, B, C, D, D + 16, None) == ERR_ALIAS
    assert f(1, 10, 64, 8, 100, A, B, C, D, C + 100 * 64 * 2 - 4, None) == ERR_ALIAS


def test_decompress_validation(ssn):
    f = ssn.lib().ssn_decompress
    assert f(1, 10, 64, 8, 100, A, B, None, D, F, None) == ERR_NULL     # ids without E
    assert f(1, 10, 64, 8, 100, A, None, C, D, F, None) == ERR_NULL     # E without ids
    assert f(1, 0, 64, 8, 100, None, None, None, None, None, None) == OK
    assert f(1, 0, 64, 8, 100, None, None, C, None, None, None) == OK   # empty ids tensor
    assert f(1, 10, 64, 8, 0, A, B, C, D, F, None) == ERR_SHAPE         # V < 1 with E
    assert f(1, 10, 64, 80, 100, A, B, C, D, F, None) == ERR_SHAPE
    assert f(1, 10, 64, 8, 100, A, B, C, D, A + 16, None) == ERR_ALIAS  # out overlaps Z
    assert f(1, 10, 64, 8, 100, A, B, C, D, F + 1, None) == ERR_ALIGN
    assert f(2, 10, 64, 8, 100, A, B, C, D, F, None) == ERR_DTYPE


def test_project_grad_validation(ssn):
    f = ssn.lib().ssn_project_grad
    assert f(1, 0, 64, 8, None, None, None, None) == OK
    assert f(1, 10, 64, 8, None, D, F, None) == ERR_NULL
    assert f(1, 10, 64, 100, A, D, F, None) == ERR_SHAPE
    assert f(1, 10, 64, 8, A, D, A + 8, None) == ERR_ALIAS


def test_project_grad_workspace_validation(ssn):
    L = ssn.lib()
    w = L.ssn_project_grad_workspace_bytes
    # up to 4 float32 partial products [N, k] where the split pays (bf16, at
    # most 16384 tokens, U of 512 KiB or more)
    assert w(1, 4096, 5120, 51, 64) == 4 * 4096 * 51 * 4
    assert w(1, 16384, 4096, 64, 64) == 4 * 16384 * 64 * 4
    assert w(1, 16385, 4096, 64, 64) == 0               # many tokens: no split
    assert w(1, 4096, 2048, 40, 48) == 0                # U of 192 KiB: no split
    assert w(0, 4096, 5120, 51, 64) == 0                # float32 storage: no split
    assert w(1, 4096, 64, 65, 65) == 0 and w(7, 4096, 4096, 64, 64) == 0
    assert w(1, 4096, 4096, 64, 63) == 0                # ldu < k
    assert ssn.project_grad_workspace_bytes(4096, 4096, 64) == 4 * 4096 * 64 * 4
    f = L.ssn_project_grad_ws
    n = 4096
    assert f(1, 0, 0, 64, 8, None, None, 8, None, None, 0, None) == OK       # N == 0 no-op
    assert f(1, 7, 10, 64, 8, A, D, 8, F, C, n, None) == ERR_DTYPE
    assert f(1, 0, 10, 64, 8, A, D, 4, F, C, n, None) == ERR_SHAPE          # ldu < k
    assert f(1, 0, 10, 64, 8, A, D, 8, F, None, n, None) == ERR_NULL        # bytes, no pointer
    assert f(1, 0, 10, 64, 8, None, D, 8, F, C, n, None) == ERR_NULL
    assert f(1, 0, 10, 64, 8, A, D, 8, F, C + 4, n, None) == ERR_ALIGN      # 16-byte aligned
    assert f(1, 0, 10, 64, 8, A, D, 8, F, A + 64, n, None) == ERR_ALIAS     # workspace on G
    assert f(1, 0, 10, 64, 8, A, D, 8, F, F - 16, n, None) == ERR_ALIAS     # workspace on GZ
    assert f(1, 0, 10, 64, 8, A, D, 8, F, D - 16, n, None) == ERR_ALIAS     # workspace on U
    assert f(1, 0, 10, 64, 8, A, D, 8, A + 8, C, n, None) == ERR_ALIAS      # GZ on G


def test_projected_table_validation(ssn):
    L = ssn.lib()
    t = L.ssn_project_table
    assert t(1, 0, 64, 8, None, None, None, None) == OK                # V == 0 no-op
    assert t(1, 100, 64, 8, None, D, F, None) == ERR_NULL
    assert t(1, 100, 64, 65, C, D, F, None) == ERR_SHAPE
    assert t(1, 100, 64, 8, C, D, C + 64, None) == ERR_ALIAS            # P overlaps E
    f = L.ssn_compress_projected
    assert f(1, 0, 64, 8, 100, None, None, None, None, None, None) == OK
    assert f(7, 10, 64, 8, 100, A, B, C, D, F, None) == ERR_DTYPE
    assert f(1, 10, 64, 8, 0, A, B, C, D, F, None) == ERR_SHAPE          # V < 1
    assert f(1, 10, 64, 8, 100, A, B, None, D, F, None) == ERR_NULL      # no table
    assert f(1, 10, 64, 8, 100, A, None, C, D, F, None) == ERR_NULL      # no ids
    assert f(1, 10, 64, 8, 100, A, B, C + 2, D, F, None) == ERR_ALIGN    # P is float32
    assert f(1, 10, 64, 8, 100, A, B, C, D, C + 100 * 8 * 4 - 4, None) == ERR_ALIAS  # Z on P
    assert f(1, 10, 64, 8, 100, A, B, C, D, A + 64, None) == ERR_ALIAS   # Z on X


def test_reparam_validation(ssn):
    L = ssn.lib()
    f = L.ssn_reparam_forward
    assert f(1, 0, 256, 128, 16, None, None, None, None, None, None) == OK
    assert f(1, 10, 256, 128, 200, A, B, C, D, F, None) == ERR_SHAPE        # k > d
    assert f(1, 10, 8, 128, 16, A, B, C, D, F, None) == ERR_SHAPE          # k > din
    assert f(1, 10, 256, 128, 16, A, None, C, D, F, None) == ERR_NULL
    assert f(1, 10, 256, 128, 16, A, B, C, D + 2, F, None) == ERR_ALIGN    # T is float32
    assert f(1, 10, 256, 128, 16, A, B, C, A + 64, F, None) == ERR_ALIAS   # T on H
    assert f(1, 10, 256, 128, 16, A, B, C, D, D + 64, None) == ERR_ALIAS   # Y on T
    w = L.ssn_reparam_workspace_bytes
    assert w(1, 32768, 14336, 64) == w(1, 32768, 14336, 64) > 0
    assert w(0, 32768, 14336, 64) == 0                                    # generic path: none
    b = L.ssn_reparam_backward
    E6 = 0x7F5000000000
    need = w(1, 1000, 256, 16)                  # 32 token splits of 32 tokens (one chunk each)
    assert need == 32 * 256 * 16 * 4
    assert b(1, 1000, 256, 128, 16, A, B, C, D, F, E6, 0x7F6000000000, 0x7F7000000000,
             need - 4, None) == ERR_SHAPE                                  # workspace too small
    assert b(1, 10, 256, 128, 16, A, B, C, D, F, E6, None, None, 0, None) == ERR_NULL
    assert b(1, 10, 256, 128, 16, A, B, C, D, F, F + 8, 0x7F7000000000, None, 0, None) == ERR_ALIAS
    e = L.ssn_factored_embedding
    assert e(1, 0, 128, 16, 100, None, None, None, None, None) == OK
    assert e(1, 10, 128, 16, 0, A, B, C, D, None) == ERR_SHAPE
    assert e(1, 10, 128, 16, 100, A, None, C, D, None) == ERR_NULL
    assert e(1, 10, 128, 16, 100, A, B + 2, C, D, None) == ERR_ALIGN      # E is float32
    assert e(1, 10, 128, 16, 100, A, B, C, B + 64, None) == ERR_ALIAS


def test_pad_basis_validation(ssn):
    f = ssn.lib().ssn_pad_basis
    assert f(1, 5120, 51, 50, A, B, None) == ERR_SHAPE              # ldu < k
    assert f(1, 5120, 0, 64, A, B, None) == ERR_SHAPE
    assert f(1, 5120, 51, 64, None, B, None) == ERR_NULL
    assert f(1, 5120, 51, 64, A, A + 64, None) == ERR_ALIAS         # the copy on top of U
    assert f(1, 5120, 51, 64, A, B + 1, None) == ERR_ALIGN
    assert f(4, 5120, 51, 64, A, B, None) == ERR_DTYPE


def test_check_ids_validation(ssn):
    f = ssn.lib().ssn_check_ids
    assert f(-1, 100, A, B, None) == ERR_SHAPE
    assert f(10, 0, A, B, None) == ERR_SHAPE                    # V >= 1
    assert f(10, 100, None, B, None) == ERR_NULL
    assert f(10, 100, A, None, None) == ERR_NULL
    assert f(0, 100, None, None, None) == ERR_NULL               # the count is always written
    assert f(10, 100, A + 2, B, None) == ERR_ALIGN
    assert f(10, 100, A, B + 4, None) == ERR_ALIGN               # int64 count
    assert f(10, 100, A, A + 8, None) == ERR_ALIAS               # count inside the id array


def test_project_weights_validation(ssn):
    L = ssn.lib()
    f = L.ssn_project_weights
    assert L.ssn_project_weights_workspace_bytes(4096, 14336, 64) == 0   # U^T W stays on chip
    assert ssn.project_weights_workspace_bytes(5120, 18432, 51) == 0
    assert f(1, 64, 0, 8, None, None, None, 0, None) == OK
    assert f(1, 64, 10, 8, None, D, None, 0, None) == ERR_NULL
    assert f(1, 64, 10, 0, A, D, None, 0, None) == ERR_SHAPE
    assert f(1, 64, -1, 8, A, D, None, 0, None) == ERR_SHAPE
    assert f(1, 4096, 10, 2048, A, D, None, 0, None) == ERR_UNSUPPORTED    # k > 1024
    assert f(1, 64, 10, 8, A, A + 64, None, 0, None) == ERR_ALIAS          # W overlaps U
    assert f(1, 64, 10, 8, A + 1, D, None, 0, None) == ERR_ALIGN
    assert f(7, 64, 10, 8, A, D, None, 0, None) == ERR_DTYPE
    g = L.ssn_project_weights_batched
    n = (ctypes.c_int64 * 2)(16, 16)
    w = (ctypes.c_void_p * 2)(A, A + 64)                                  # overlapping matrices
    assert g(1, 2, 64, n, 8, w, D, None) == ERR_ALIAS
    assert g(1, 0, 64, n, 8, w, D, None) == ERR_SHAPE
    assert g(1, 17, 64, n, 8, w, D, None) == ERR_SHAPE
    assert g(1, 2, 64, None, 8, w, D, None) == ERR_NULL
    n0 = (ctypes.c_int64 * 2)(0, 0)
    assert g(1, 2, 64, n0, 8, w, None, None) == OK                        # all empty: no-op


def test_sparta_validation(ssn):
    L = ssn.lib()
    P = ctypes.c_void_p
    s = L.ssn_sparta_snapshot
    assert s(100, 0, None, 0, None, None, None) == OK                       # empty round
    assert s(100, 10, None, 95, A, B, None) == ERR_SHAPE                    # segment past n
    assert s(100, 10, None, -1, A, B, None) == ERR_SHAPE
    assert s(0, 10, C, 0, A, B, None) == ERR_SHAPE                          # list on empty theta
    assert s(100, 10, None, 0, None, B, None) == ERR_NULL
    assert s(100, 10, None, 0, A + 2, B, None) == ERR_ALIGN
    assert s(100, 10, C + 4, 0, A, B, None) == ERR_ALIGN                    # int64 positions
    assert s(100, 10, None, 0, A, A + 64, None) == ERR_ALIAS                # snap inside theta
    assert s(100, 10, C, 0, A, C + 8, None) == ERR_ALIAS                    # snap on the positions
    a = L.ssn_sparta_average
    cs = (P * 2)(A, B)
    ds = (P * 2)(C, D)
    w = (ctypes.c_float * 2)(1.0, 3.0)
    assert a(0, 10, cs, None, F, ds, None) == ERR_SHAPE
    assert a(65, 10, cs, None, F, ds, None) == ERR_SHAPE
    assert a(2, 0, None, w, None, None, None) == OK
    assert a(2, 10, cs, (ctypes.c_float * 2)(1.0, -1.0), F, ds, None) == ERR_SHAPE   # negative
    assert a(2, 10, cs, (ctypes.c_float * 2)(0.0, 0.0), F, ds, None) == ERR_SHAPE    # zero sum
    assert a(2, 10, cs, (ctypes.c_float * 2)(1.0, float("nan")), F, ds, None) == ERR_SHAPE
    assert a(2, 10, (P * 2)(A, None), w, F, ds, None) == ERR_NULL
    assert a(2, 10, cs, w, F + 2, ds, None) == ERR_ALIGN
    assert a(2, 10, cs, w, A + 8, ds, None) == ERR_ALIAS                    # acc on a chunk
    assert a(2, 10, cs, w, F, (P * 2)(C, B), None) == ERR_ALIAS             # delta on a chunk
    assert a(2, 10, cs, w, F, (P * 2)(C, C + 8), None) == ERR_ALIAS         # deltas overlap
    assert a(2, 10, cs, w, F, (P * 2)(F + 4, None), None) == ERR_ALIAS      # delta on acc
    d = L.ssn_delta_rule
    assert d(100, 0, None, 0, None, None, None, 1.0, None) == OK
    assert d(100, 10, None, 91, A, B, C, 1.0, None) == ERR_SHAPE
    assert d(100, 10, None, 0, A, B, C, float("inf"), None) == ERR_SHAPE    # lambda finite
    assert d(100, 10, None, 0, A, None, C, 1.0, None) == ERR_NULL
    assert d(100, 10, None, 0, A, B + 1, C, 1.0, None) == ERR_ALIGN
    assert d(100, 10, None, 0, A, A + 40, C, 1.0, None) == ERR_ALIAS        # avg inside theta
    assert d(100, 10, None, 0, A, B, A + 396, 1.0, None) == ERR_ALIAS       # snap overlaps theta's end


def test_sparta_segments_tile_and_rotate(ssn):
    """Host logic of the rotation (ssn_sparta_segment) against the oracle's
    schedule: 20 contiguous segments tile [0, n) for any n, sizes differ by
    at most one, and round r takes segment r mod 20."""
    from oracle import ssn_oracle as O
    for n in (0, 1, 19, 20, 21, 1000, 320_000_003, (1 << 56) - 5):
        seen = 0
        sizes = []
        for r in range(ssn.SPARTA_SEGMENTS):
            first, m = ssn.sparta_segment(n, r)
            assert (first, m) == O.sparta_segment(n, r, ssn.SPARTA_SEGMENTS)
            assert first == seen
            seen += m
            sizes.append(m)
            assert ssn.sparta_segment(n, r + 3 * ssn.SPARTA_SEGMENTS) == (first, m)
        assert seen == n
        assert max(sizes) - min(sizes) <= 1
    for n, r, S in [(10, 3, 4), (999, 7, 7), (12345, 11, 1000)]:
        assert ssn.sparta_segment(n, r, S) == O.sparta_segment(n, r, S)
    L = ssn.lib()
    f, m = ctypes.c_int64(), ctypes.c_int64()
    assert L.ssn_sparta_segment(-1, 0, 20, ctypes.byref(f), ctypes.byref(m)) == ERR_SHAPE
    assert L.ssn_sparta_segment(10, -1, 20, ctypes.byref(f), ctypes.byref(m)) == ERR_SHAPE
    assert L.ssn_sparta_segment(10, 0, 0, ctypes.byref(f), ctypes.byref(m)) == ERR_SHAPE
    assert L.ssn_sparta_segment(10, 0, 20, None, ctypes.byref(m)) == ERR_NULL


def test_binding_refuses_cpu_tensors_and_missing_library(ssn, monkeypatch):
    import torch
    x = torch.zeros(4, 64, dtype=torch.bfloat16)
    ids = torch.zeros(4, dtype=torch.int32)
    with pytest.raises(ValueError, match="GPU tensor"):
        ssn.compress(x, ids, x, torch.zeros(64, 8, dtype=torch.bfloat16))
    monkeypatch.setattr(ssn, "_lib", None)
    monkeypatch.setattr(ssn, "LIB_PATH", "/nonexistent/libssn.so")
    with pytest.raises(RuntimeError, match="not built"):
        ssn.lib()
