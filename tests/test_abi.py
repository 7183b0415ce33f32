"""The C-ABI library loads, exports every function include/dvs.h declares, and
rejects bad arguments on the host (no GPU needed: nothing is launched)."""
import ctypes
import os
import re

import pytest

from paper_2609_26638_amd import dvs

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "dvs.h")

needs_lib = pytest.mark.skipif(not os.path.exists(dvs.LIB_PATH),
                               reason="libdvs.so not built (run __graft_entry__.build())")


def _declared():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?[\w\s\*]+?\b(\w+)\s*\(", src, flags=re.M)))


def test_header_declares_the_hot_path():
    names = _declared()
    for n in ("attn_hybrid_block", "argmax_accept", "kv_commit", "dvs_attn_workspace_bytes",
              "dvs_last_error", "dvs_version"):
        assert n in names


@needs_lib
def test_every_declared_symbol_is_exported():
    lib = ctypes.CDLL(dvs.LIB_PATH)
    for n in _declared():
        assert hasattr(lib, n), n
    assert set(_declared()) <= set(dvs.EXPORTED)


@needs_lib
def test_version_and_workspace_query():
    L = dvs.lib()
    assert L.dvs_version() >= 100
    b = dvs.attn_workspace_bytes(64, 32, 32, 16, 4, 128, 1042, 2048, dvs.DVS_BF16)
    assert b > 0 and b % 256 == 0
    assert dvs.attn_workspace_bytes(0, 32, 32, 16, 4, 128, 1042) == 0
    assert dvs.attn_workspace_bytes(4, 1, 0, 6, 4, 128, 10) == 0       # Hq % Hkv != 0


@needs_lib
def test_host_validation_rejects_bad_arguments():
    L = dvs.lib()
    nul = None
    fake = ctypes.c_void_p(0x1000)   # never dereferenced: validation fails first
    rc = L.attn_hybrid_block(nul, nul, nul, nul, nul, nul, nul, 1, 1, 1, 4, 4, 64, 4, 4, 0.1,
                             0, 0, nul, nul, nul, 0, nul)
    assert rc == -1 and b"NULL" in L.dvs_last_error()
    args = [fake] * 7
    rc = L.attn_hybrid_block(*args, 1, 2, 2, 6, 4, 64, 4, 4, 0.1, 1, 0, fake, nul, fake, 1 << 30, nul)
    assert rc == -1                                   # Hq % Hkv
    rc = L.attn_hybrid_block(*args, 1, 2, 2, 4, 4, 80, 4, 4, 0.1, 1, 0, fake, nul, fake, 1 << 30, nul)
    assert rc == -2                                   # head_dim 80 unsupported
    rc = L.attn_hybrid_block(*args, 1, 2, 2, 4, 4, 64, 4, 4, 0.1, 7, 0, fake, nul, fake, 1 << 30, nul)
    assert rc == -2                                   # dtype
    rc = L.attn_hybrid_block(*args, 1, 2, 2, 4, 4, 64, 4, 4, 0.1, 1, 100, fake, nul, fake, 1 << 30, nul)
    assert rc == -1                                   # chunk not a multiple of 64
    rc = L.attn_hybrid_block(*args, 1, 2, 2, 4, 4, 64, 4, 4, 0.1, 1, 0, fake, nul, fake, 16, nul)
    assert rc == -4                                   # workspace too small
    rc = L.argmax_accept(fake, 1, 2, 4, 100, 5, fake, 4, fake, fake, nul, nul)
    assert rc == -1                                   # n_causal > R
    rc = L.argmax_accept(fake, 1, 2, 4, 100, 3, fake, 1, fake, fake, nul, nul)
    assert rc == -1                                   # draft narrower than n_causal-1
    rc = L.kv_commit(2000, 2, 2, *([fake] * 5), 4, fake, fake, 8, fake, fake, 1, fake, fake, 8,
                     -1, fake, nul, nul)
    assert rc == -1                                   # S > 1024
    rc = L.kv_commit(2, 4, 2, *([fake] * 5), 4, fake, fake, 8, fake, fake, 3, fake, fake, 8,
                     -1, fake, nul, nul)
    assert rc == -1                                   # mask rows fewer than the draft width


@needs_lib
def test_noalloc_rejects_oversized_shape_before_any_hip_call():
    """attn_hybrid_block_noalloc checks the shape against its scratch array
    first: an oversized call fails on the host, with nothing launched."""
    L = dvs.lib()
    fake = ctypes.c_void_p(0x1000)
    # 64 sequences, 64 rows, aligned 64-key chunks over 1030 pages: > 64 MiB
    rc = L.attn_hybrid_block_noalloc(*([fake] * 7), 64, 32, 32, 16, 4, 128, 1030, 8, 0.1, 1, 64,
                                     fake, None, None)
    assert rc == -4 and b"scratch" in L.dvs_last_error()
    rc = L.attn_hybrid_block_noalloc(*([fake] * 7), 1, 2, 2, 6, 4, 64, 4, 4, 0.1, 1, 0, fake,
                                     None, None)
    assert rc == -1                                   # Hq % Hkv (checked before the device lookup)
