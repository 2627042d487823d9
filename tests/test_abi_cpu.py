"""The C-ABI library loads, exports what include/kvs.h declares, and rejects
bad arguments before touching the GPU (no GPU needed)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "kvs.h")
LIB = os.path.join(ROOT, "paper_2609_35750_amd", "libkvs.so")

pytestmark = pytest.mark.skipif(not os.path.exists(LIB), reason="libkvs.so not built (run __graft_entry__.build())")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(kvs_[a-z0-9_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def kvs():
    from paper_2609_35750_amd import kvs as k

    return k


def test_every_declared_symbol_is_exported():
    lib = ctypes.CDLL(LIB)
    names = declared_functions()
    assert len(names) >= 14
    for n in names:
        assert hasattr(lib, n), n


def test_binding_covers_every_symbol(kvs):
    assert set(declared_functions()) <= set(kvs.SIGNATURES)


def test_version_and_strings(kvs):
    assert kvs.lib.kvs_abi_version() == 3
    for s in range(10):
        assert kvs.lib.kvs_status_string(s)
    assert kvs.lib.kvs_status_string(99) == b"unknown status"


FAKE = 1 << 20  # 16-byte aligned, never dereferenced: validation fails first


def _fwd(kvs, B=1, T=64, Hq=4, Hkv=2, D=64, q=FAKE, ws=FAKE, ws_bytes=1 << 20, scale=0.125, ev=FAKE):
    return kvs.lib.kvs_evict_attn_fwd(q, FAKE, FAKE, ev, FAKE, FAKE, B, T, Hq, Hkv, D, scale, ws, ws_bytes, None)


def test_forward_validation(kvs):
    assert _fwd(kvs, Hq=6, Hkv=4) == kvs.KVS_ERR_SHAPE
    assert _fwd(kvs, D=96) == kvs.KVS_ERR_SHAPE
    assert _fwd(kvs, B=0) == kvs.KVS_ERR_SHAPE
    assert _fwd(kvs, T=0) == kvs.KVS_ERR_SHAPE
    assert _fwd(kvs, q=None) == kvs.KVS_ERR_NULL
    assert _fwd(kvs, ev=None) == kvs.KVS_ERR_NULL
    assert _fwd(kvs, q=FAKE + 2) == kvs.KVS_ERR_ALIGN
    assert _fwd(kvs, ws=FAKE + 16) == kvs.KVS_ERR_ALIGN
    assert _fwd(kvs, ws_bytes=8) == kvs.KVS_ERR_WORKSPACE
    assert _fwd(kvs, ws=None) == kvs.KVS_ERR_NULL
    assert _fwd(kvs, scale=0.0) == kvs.KVS_ERR_SHAPE
    assert _fwd(kvs, T=(1 << 20) + 1) == kvs.KVS_ERR_UNSUPPORTED
    assert _fwd(kvs, Hq=130, Hkv=1) == kvs.KVS_ERR_UNSUPPORTED
    assert b"multiple" in kvs.lib.kvs_last_error() or True


def test_backward_and_varlen_validation(kvs):
    L = kvs.lib
    need = L.kvs_evict_attn_bwd_workspace(1, 64, 4, 2, 64)
    assert need > L.kvs_evict_attn_fwd_workspace(1, 64, 4, 2, 64) > 0
    st = L.kvs_evict_attn_bwd(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None, FAKE, FAKE,
                              1, 64, 4, 2, 64, 0.125, FAKE, need, None)
    assert st == kvs.KVS_ERR_NULL
    st = L.kvs_evict_attn_bwd(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE,
                              1, 64, 4, 2, 64, 0.125, FAKE, need - 1, None)
    assert st == kvs.KVS_ERR_WORKSPACE
    st = L.kvs_evict_attn_varlen_fwd(FAKE, FAKE, FAKE, FAKE, None, FAKE, FAKE, 2, 100, 60, 4, 2, 64, 0.1,
                                     FAKE, 1 << 20, None)
    assert st == kvs.KVS_ERR_NULL
    st = L.kvs_evict_attn_varlen_bwd(FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE,
                                     2, 100, 60, 4, 3, 64, 0.1, FAKE, 1 << 20, None)
    assert st == kvs.KVS_ERR_SHAPE


def test_ex_validation(kvs):
    """The *_ex calls: the fixed layout needs Ntot = B * max_seqlen, unknown flag bits are refused,
    and every other check is that of the plain calls."""
    L = kvs.lib
    fwd_ex = lambda cu, B, N, T, flags, ws_bytes=1 << 20: L.kvs_evict_attn_fwd_ex(
        FAKE, FAKE, FAKE, FAKE, cu, FAKE, FAKE, B, N, T, 4, 2, 64, 0.125, flags, FAKE, ws_bytes, None)
    assert fwd_ex(None, 2, 100, 60, 0) == kvs.KVS_ERR_SHAPE          # 100 != 2 * 60
    assert fwd_ex(None, 2, 120, 60, 4) == kvs.KVS_ERR_UNSUPPORTED     # unknown bit
    assert fwd_ex(FAKE, 2, 100, 60, 1 << 31) == kvs.KVS_ERR_UNSUPPORTED
    assert fwd_ex(None, 2, 120, 60, 3, ws_bytes=8) == kvs.KVS_ERR_WORKSPACE
    need = L.kvs_evict_attn_bwd_workspace(2, 60, 4, 2, 64)
    bwd_ex = lambda cu, flags, dq=FAKE, ws_bytes=need: L.kvs_evict_attn_bwd_ex(
        FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, cu, dq, FAKE, FAKE, 2, 120, 60, 4, 2, 64, 0.125, flags, FAKE,
        ws_bytes, None)
    assert bwd_ex(None, 8) == kvs.KVS_ERR_UNSUPPORTED
    assert bwd_ex(None, 1, dq=None) == kvs.KVS_ERR_NULL
    assert bwd_ex(None, 2, ws_bytes=need - 1) == kvs.KVS_ERR_WORKSPACE
    assert kvs.FLAG_NO_EMPTY_SKIP == 1 and kvs.FLAG_FULL_AS_PARTIAL == 2


def test_empty_batch_is_a_no_op(kvs):
    """Ntot = 0 (varlen traces that are all empty) returns OK without looking at any tensor
    pointer or the workspace, so those may be NULL (cu_seqlens, B + 1 entries, is still required);
    shapes, scale and flags are still checked.
    No HIP call happens, so this runs without a GPU."""
    L = kvs.lib
    fwd = lambda scale=0.125, Hq=4, D=64: L.kvs_evict_attn_varlen_fwd(
        None, None, None, None, FAKE, None, None, 3, 0, 1, Hq, 2, D, scale, None, 0, None)
    assert fwd() == kvs.KVS_OK
    assert fwd(scale=float("nan")) == kvs.KVS_ERR_SHAPE
    assert fwd(Hq=3) == kvs.KVS_ERR_SHAPE
    assert fwd(D=96) == kvs.KVS_ERR_SHAPE
    st = L.kvs_evict_attn_varlen_bwd(None, None, None, None, None, None, None, FAKE, None, None, None,
                                     3, 0, 1, 4, 2, 128, 0.1, None, 0, None)
    assert st == kvs.KVS_OK
    st = L.kvs_evict_attn_fwd_ex(None, None, None, None, None, None, None, 2, 0, 1, 4, 2, 64, 0.1, 3, None, 0, None)
    assert st == kvs.KVS_ERR_SHAPE                                  # fixed layout: Ntot = B * max_seqlen
    st = L.kvs_evict_attn_bwd_ex(None, None, None, None, None, None, None, None, None, None, None,
                                 2, 0, 1, 4, 2, 64, 0.1, 4, None, 0, None)
    assert st != kvs.KVS_OK
    st = L.kvs_evict_attn_fwd_noalloc(None, None, None, None, FAKE, None, None, 2, 0, 1, 4, 2, 64, 0.1, None)
    assert st == kvs.KVS_OK


def test_noalloc_forward_validation(kvs):
    """The allocation-free forward refuses problems beyond its scratch before any HIP call."""
    L = kvs.lib
    call = lambda cu, B, N, T, Hq=4, Hkv=2, D=64: L.kvs_evict_attn_fwd_noalloc(
        FAKE, FAKE, FAKE, FAKE, cu, FAKE, FAKE, B, N, T, Hq, Hkv, D, 0.125, None)
    # 32768 key tiles of statistics at most: B + Ntot / 64 + 2
    assert call(FAKE, 4, 2_200_000, 1 << 20) == kvs.KVS_ERR_UNSUPPORTED
    assert b"scratch" in L.kvs_last_error()
    assert call(None, 2, 100, 60) == kvs.KVS_ERR_SHAPE          # fixed layout: Ntot = B * max_seqlen
    assert call(None, 2, 120, 60, Hq=6, Hkv=4) == kvs.KVS_ERR_SHAPE
    st = L.kvs_evict_attn_fwd_noalloc(None, FAKE, FAKE, FAKE, None, FAKE, FAKE, 2, 120, 60, 4, 2, 64, 0.125, None)
    assert st == kvs.KVS_ERR_NULL


def test_classify_and_check_validation(kvs):
    L = kvs.lib
    assert L.kvs_classify_tiles(FAKE, None, 1, 100, 20, 64, FAKE, None) == kvs.KVS_ERR_SHAPE
    assert L.kvs_classify_tiles(FAKE, None, 1, 100, 64, 48, FAKE, None) == kvs.KVS_ERR_SHAPE
    assert L.kvs_classify_tiles(None, None, 1, 100, 64, 64, FAKE, None) == kvs.KVS_ERR_NULL
    assert L.kvs_check_evict_at(FAKE, None, 1, 10, None, None) == kvs.KVS_ERR_NULL
    lens = (ctypes.c_int32 * 3)(100, 0, 65)
    assert L.kvs_classify_tiles_size(lens, 3, 32, 64) == 4 * 2 + 0 + 3 * 2


def test_prof_read_without_records(kvs):
    kvs.kvs_prof_reset()
    assert kvs.kvs_prof_read("fwd") == (0, 0.0)


def test_bench_probe_is_outside_the_library(kvs):
    """The matrix-core probe lives in the benchmark's own library, not in the libkvs ABI."""
    assert not hasattr(ctypes.CDLL(LIB), "kvs_measure_mfma_rate")
    probe = os.path.join(ROOT, "paper_2609_35750_amd", "libkvs_bench.so")
    lib = ctypes.CDLL(probe)
    lib.kvs_bench_mfma_rate.argtypes = [ctypes.c_void_p, ctypes.c_void_p]
    assert lib.kvs_bench_mfma_rate(None, None) == 1   # NULL result pointer, before any HIP call
