"""The C ABI: every function declared in include/pace.h is exported by libpace.so, the
host-only helpers agree with the oracle, and bad arguments are rejected before any launch
(these calls never reach the GPU, so they run on the CPU)."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "pace.h")

pace = pytest.importorskip("paper_2608_27206_amd.pace")
if not os.path.exists(pace.LIB_PATH):
    pytest.skip("libpace.so not built", allow_module_level=True)


def declared_functions():
    txt = open(HEADER).read()
    txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
    return sorted(set(re.findall(r"\b(pace_[a-z0-9_]+)\s*\(", txt)))


def test_every_declared_symbol_is_exported():
    L = ctypes.CDLL(pace.LIB_PATH)
    names = declared_functions()
    assert len(names) >= 15
    for n in names:
        assert hasattr(L, n), f"{n} declared in pace.h but not exported"


def test_binding_covers_header():
    assert sorted(pace.EXPORTED) == declared_functions()


def test_keep_count_matches_oracle():
    from oracle import ddae
    for r in (0.05, 0.1, 0.2, 0.25, 1.0, 0.0):
        for n in list(range(0, 300)) + [10549, 42196]:
            assert pace.keep_count(r, n) == ddae.keep_count(r, n)
    assert pace.keep_count(0.1, -1) == -1


def test_keep_from_density_matches_oracle():
    from oracle import ddae
    for rho in (0.0, 0.2, 0.371, 0.5, 0.9999, 1.0, 1.3, -0.2):
        for n in (1, 37, 256, 2304, 10549):
            assert pace.keep_from_density(rho, n) == ddae.keep_from_density(rho, n)
    assert pace.keep_from_density(0.5, 100) == 15
    assert pace.lib().pace_keep_from_density(0.5, 0.3, 0.2, 10) == -1


def test_target_size_matches_oracle():
    from oracle import apc
    cases = [(0.25, 1120, 1680, 0, 1e12, 28), (0.9, 2000, 2000, 0, 1e6, 1), (0.0, 1000, 1000, 250000, 1e12, 1),
             (1.0, 50, 50, 0, 1e12, 28), (0.37, 2156, 3836, 256 * 784, 2048 * 784, 28),
             (0.6, 3836, 2156, 0, 1e12, 1), (0.5, 30, 10, 0, 1e12, 28)]
    for c in cases:
        assert pace.apc_target_size(*c) == apc.target_size(*c), c


def _status(fn, *args):
    return getattr(pace.lib(), fn)(*args)


def test_errors_before_launch():
    L = pace.lib()
    fake = ctypes.c_void_p(0x1000)   # aligned, never dereferenced: validation fails first
    # null pointers
    st = L.pace_vit_attention(None, None, None, 10, 2, 80, None, 1, 10, 0.1, None, None, None, None, 0, None)
    assert st == 1 and "null" in L.pace_last_error().decode()
    # unsupported head dim
    st = L.pace_vit_attention(fake, fake, fake, 10, 2, 64, fake, 1, 10, 0.1, fake, None, None, None, 0, None)
    assert st == 2 and "head dim" in L.pace_last_error().decode()
    # misaligned
    st = L.pace_vit_attention(ctypes.c_void_p(0x1002), fake, fake, 10, 2, 80, fake, 1, 10, 0.1, fake,
                              None, None, None, 0, None)
    assert st == 1
    # max_seglen above N
    st = L.pace_vit_attention(fake, fake, fake, 10, 2, 80, fake, 1, 11, 0.1, fake, None, None, None, 0, None)
    assert st == 1
    # mass without lse or workspace
    st = L.pace_vit_attention(fake, fake, fake, 10, 2, 80, fake, 1, 10, 0.1, fake, None, fake, None, 0, None)
    assert st == 3
    # a long segment at head dim 80 needs the workspace for its V^T tiles
    st = L.pace_vit_attention(fake, fake, fake, 2048, 2, 80, fake, 1, 2048, 0.1, fake, fake, None, None, 0, None)
    assert st == 3 and "workspace" in L.pace_last_error().decode()
    # GQA heads not divisible
    st = L.pace_prefill_attention_with_mass(fake, fake, fake, 10, 6, 4, 128, fake, 1, 10, None, fake, fake, 5,
                                            5, fake, fake, 5, 0.1, fake, fake, fake, None, 0, None)
    assert st == 1
    # K > N in DDAE selection
    nv = (ctypes.c_int * 1)(10)
    kk = (ctypes.c_int * 1)(11)
    st = L.pace_ddae_select_varlen(fake, 1, 1, None, fake, 1, 1, nv, kk, 0, 0.5, 0.5, None, 0, fake,
                                   None, None, None, fake, 1 << 20, None)
    assert st == 1 and "K=11" in L.pace_last_error().decode()
    # an image without tokens
    nv0 = (ctypes.c_int * 1)(0)
    k0 = (ctypes.c_int * 1)(0)
    st = L.pace_ddae_select_varlen(fake, 1, 1, None, fake, 1, 1, nv0, k0, 0, 0.5, 0.5, None, 0, fake,
                                   None, None, None, fake, 1 << 20, None)
    assert st == 1 and "0 tokens" in L.pace_last_error().decode()
    # bad mode, tau
    kk[0] = 3
    st = L.pace_ddae_select_varlen(fake, 1, 1, None, fake, 1, 1, nv, kk, 2, 0.5, 0.5, None, 0, fake,
                                   None, None, None, fake, 1 << 20, None)
    assert st == 1
    st = L.pace_ddae_select_varlen(fake, 1, 1, None, fake, 1, 1, nv, kk, 0, 0.0, 0.5, None, 0, fake,
                                   None, None, None, fake, 1 << 20, None)
    assert st == 1
    # workspace too small
    st = L.pace_ddae_select_varlen(fake, 1, 1, None, fake, 1, 1, nv, kk, 0, 0.5, 0.5, None, 0, fake,
                                   None, None, None, fake, 16, None)
    assert st == 3
    # row_bytes not a multiple of 16
    st = L.pace_topk_gather(fake, 10, 3, fake, 24, fake, fake, None, 0, None)
    assert st == 1
    # APC: image not a multiple of the patch, patch too large, upsampling
    st = L.pace_apc_density(fake, 100, 98, 14, 0.1, 0.6, 1.5, None, fake, fake, 1 << 30, None)
    assert st == 1
    st = L.pace_apc_density(fake, 68, 68, 17, 0.1, 0.6, 1.5, None, fake, fake, 1 << 30, None)
    assert st == 1
    st = L.pace_apc_downsample(fake, 10, 10, fake, 11, 10, None)
    assert st == 1
    # APC on embeddings: empty, odd address, workspace too small
    st = L.pace_apc_density_features(fake, 100, 0, 0.1, 0.6, 1.5, None, fake, fake, 1 << 30, None)
    assert st == 1
    st = L.pace_apc_density_features(ctypes.c_void_p(0x1001), 100, 16, 0.1, 0.6, 1.5, None, fake, fake,
                                     1 << 30, None)
    assert st == 1
    st = L.pace_apc_density_features(fake, 100, 16, 0.1, 0.6, 1.5, None, fake, fake, 16, None)
    assert st == 3


def test_workspace_sizes_monotone():
    L = pace.lib()
    assert L.pace_apc_density_workspace_size(2156, 3836, 14) > L.pace_apc_density_workspace_size(448, 448, 14)
    assert L.pace_ddae_select_workspace_size(10549, 1) >= 3 * 10549 * 4
    assert L.pace_vit_attention_workspace_size(42196, 16, 80, 700, 64) == 42196 * 16 * 4
    cols = 64 * ((42196 + 63) // 64) + 64          # V^T columns: segments start on 64-column boundaries
    vt = (16 * 81 * cols * 2 + 255) // 256 * 256
    lse = (42196 * 16 * 4 + 255) // 256 * 256
    assert L.pace_vit_attention_workspace_size(42196, 16, 80, 1, 42196) == lse + vt + 1 * 16 * 4
    assert L.pace_vit_attention_workspace_size(42196, 16, 128, 1, 42196) == 42196 * 16 * 4


def test_noalloc_select_rejects_more_than_its_scratch():
    """The allocation-free selection refuses, before touching the GPU, a batch whose scratch would
    exceed the static 4 MiB; bad counts are refused the same way."""
    L = pace.lib()
    cap = L.pace_ddae_select_noalloc_max_bytes()
    assert cap == 4 << 20
    big = 400000
    assert L.pace_ddae_select_workspace_size(big, 1) > cap >= L.pace_ddae_select_workspace_size(300000, 1)
    one = (ctypes.c_int * 1)
    null = None
    st = L.pace_ddae_select_varlen_noalloc(null, 16, 4, null, null, 28, 1, one(big), one(10), 0, 0.5, 0.5,
                                           null, 0, null, null, null, null, null)
    assert st == 3 and b"static scratch" in L.pace_last_error()
    st = L.pace_ddae_select_varlen_noalloc(null, 16, 4, null, null, 28, 1, one(0), one(0), 0, 0.5, 0.5,
                                           null, 0, null, null, null, null, null)
    assert st == 1
    st = L.pace_ddae_select_varlen_noalloc(null, 16, 4, null, null, 28, 0, one(5), one(1), 0, 0.5, 0.5,
                                           null, 0, null, null, null, null, null)
    assert st == 1
