"""libslim loads, exports every entry point of include/slim.h, and rejects bad arguments on the
host before touching a GPU (no compute call here needs a device)."""
import ctypes
import re

import pytest

from paper_2608_24070_amd import slim

A = 1 << 20          # a fake, 16-byte aligned, non-null "device" address (never dereferenced)
MIS = A + 4          # misaligned


def test_library_exports_every_declared_symbol():
    lib = slim.lib()
    syms = slim.header_symbols()
    assert {"slim_pack", "slim_pack_bwd", "slim_linear", "slim_linear_bwd_dx", "slim_linear_workspace",
            "slim_bwd_dx_workspace", "slim_workspace_init", "slim_status_string", "slim_abi_version",
            "slim_timing_enable", "slim_timing_reset", "slim_timing_read", "slim_pack_adapter"} <= set(syms)
    for name in syms:
        assert hasattr(lib, name), name


def test_version_and_status_strings():
    assert slim.slim_abi_version() == 2
    for code in range(10):
        assert slim.status_string(code).startswith("SLIM_")
    assert "unknown" in slim.status_string(99)


def test_pack_validation():
    ok = dict(W=A, N=16, K=128, codes=A, meta=A, scales=A, mask=None, stream=None)
    def call(**kw):
        a = dict(ok, **kw)
        return slim.slim_pack(a["W"], a["N"], a["K"], a["codes"], a["meta"], a["scales"], a["mask"], a["stream"])
    assert call(W=None) == 1
    assert call(codes=None) == 1
    assert call(K=100) == 2
    assert call(K=64) == 2
    assert call(N=0) == 2
    assert call(N=8) == 2           # whole 16-row blocks
    assert call(N=40) == 2
    assert call(W=MIS) == 4
    assert call(mask=MIS) == 4


def test_pack_bwd_validation():
    def call(N=128, K=256, codes=A, codesT=A, mask=None):
        return slim.slim_pack_bwd(codes, A, A, N, K, codesT, A, A, mask, None)
    assert call(codes=None) == 1
    assert call(N=24) == 2          # N % 128: the transposed pack chunks N by 128
    assert call(N=64) == 2
    assert call(K=200) == 2
    assert call(codesT=MIS) == 4


def test_pack_adapter_validation():
    assert slim.slim_pack_adapter(None, A, 128, 64, 16, A, A, None) == 1
    assert slim.slim_pack_adapter(A, A, 128, 64, 24, A, A, None) == 2
    assert slim.slim_pack_adapter(A, A, 128, 64, 16, MIS, A, None) == 4


def test_linear_validation_and_workspace():
    need = slim.slim_linear_workspace(16, 512, 512, 32)
    assert need > 0
    def call(X=A, xdt=1, M=16, N=512, K=512, L=A, R=A, r=32, Y=A, ws=A, wsb=None):
        return slim.slim_linear(X, xdt, M, N, K, A, A, A, L, R, r, Y, ws, need if wsb is None else wsb, None)
    assert call(X=None) == 1
    assert call(L=None) == 1                  # r > 0 needs both factors
    assert call(r=0) == 1                     # r == 0 needs both NULL
    assert call(xdt=2) == 3
    assert call(N=500) == 2
    assert call(K=500) == 2
    assert call(r=24) == 2
    assert call(M=0) == 2
    assert call(X=MIS) == 4
    assert call(wsb=need - 1) == slim.SLIM_EWORKSPACE
    assert call(ws=None) == slim.SLIM_EWORKSPACE


def test_bwd_workspace_and_shape_rules():
    assert slim.slim_bwd_dx_workspace(16, 28672, 8192, 512) > 0
    with pytest.raises(slim.SlimError):
        slim.slim_bwd_dx_workspace(16, 1040, 512, 0)      # backward needs N % 128
    def call(N=1024, K=512, r=0):
        return slim.slim_linear_bwd_dx(A, 1, 4, N, K, A, A, A, None, None, r, A, A, 1 << 30, None)
    assert call(N=1040) == 2


def test_sizes_past_32bit_offsets_are_refused():
    # large M: the reduction at most 2^23 and M r, rows r below 2^30 (32-bit buffer offsets);
    # small M has no such limit
    big = (1 << 23) + 128
    assert slim.slim_linear_workspace(16, 16, big, 0) > 0
    assert slim.slim_linear_workspace(64, 16, 1 << 23, 0) > 0
    with pytest.raises(slim.SlimError):
        slim.slim_linear_workspace(64, 16, big, 0)
    with pytest.raises(slim.SlimError):
        slim.slim_bwd_dx_workspace(64, big, 128, 0)                # backward reduction is N
    assert slim.slim_linear_workspace(1 << 21, 16, 128, 256) > 0
    with pytest.raises(slim.SlimError):
        slim.slim_linear_workspace(1 << 21, 16, 128, 512)          # M r = 2^30
    with pytest.raises(slim.SlimError):
        slim.slim_linear_workspace(64, 1 << 21, 128, 512)          # N r = 2^30
    assert slim.slim_linear(A, 1, 64, 16, big, A, A, A, None, None, 0, A, A, 1 << 30, None) == slim.SLIM_EUNSUPPORTED


@pytest.mark.parametrize("M,N,K,r", [(1, 4096, 4096, 384), (16, 4096, 4096, 384), (2048, 11008, 4096, 384),
                                     (8192, 28672, 8192, 512), (4096, 5120, 13824, 512)])
def test_workspace_sizes_are_modest(M, N, K, r):
    fwd = slim.slim_linear_workspace(M, N, K, r)
    bwd = slim.slim_bwd_dx_workspace(M, N, K, r)
    out_bytes = 4 * M * max(N, K)
    assert fwd < 64 * 2 ** 20 + out_bytes
    assert bwd < 64 * 2 ** 20 + out_bytes


COUNTER_REGION = 4096 * 4    # the workspace's leading counter region (SLIM_COUNTER_SLOTS words)


@pytest.mark.parametrize("M,N,K,r", [(1, 16, 128, 0), (1, 16, 128, 16), (16, 4096, 4096, 384), (33, 256, 256, 16)])
def test_workspace_holds_counter_region_and_data(M, N, K, r):
    # the data regions (adapter intermediate, partials) follow the counter region
    assert slim.slim_linear_workspace(M, N, K, r) >= COUNTER_REGION + (2 * M * r if r else 0)
    if N % 128 == 0:
        assert slim.slim_bwd_dx_workspace(M, N, K, r) >= COUNTER_REGION + (2 * M * r if r else 0)


def test_workspace_init_requires_counter_region():
    assert slim.slim_workspace_init(A, COUNTER_REGION - 4, None) == slim.SLIM_EWORKSPACE   # before any GPU call


def test_binding_constants_match_header_enums():
    text = open(slim.HEADER).read()
    enums = dict((k, int(v)) for k, v in re.findall(r"\b(SLIM_[A-Z0-9]+)\s*=\s*(\d+)", text))
    assert len(enums) == 13
    for name, value in enums.items():
        assert getattr(slim, name) == value, name
    assert int(re.search(r"#define SLIM_ABI_VERSION (\d+)", text).group(1)) == slim.slim_abi_version()


def test_noalloc_refuses_sizes_past_its_scratch_before_touching_a_device():
    # a 5120 x 5120 layer at M = 4096 needs 76 MiB of workspace, more than the 64 MiB scratch
    assert slim.slim_linear_workspace(4096, 5120, 5120, 512) > slim.SLIM_NOALLOC_SCRATCH_BYTES
    assert slim.slim_linear_noalloc(A, 1, 4096, 5120, 5120, A, A, A, A, A, 512, A, None) == slim.SLIM_EWORKSPACE
    # argument errors are reported the same way as by slim_linear
    assert slim.slim_linear_noalloc(A, 1, 16, 100, 512, A, A, A, None, None, 0, A, None) == slim.SLIM_ESHAPE
    assert "noalloc" in " ".join(slim.header_symbols())
