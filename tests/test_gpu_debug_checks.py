"""PACE_DEBUG=1: device-side metadata is copied to the host and checked before any launch, so
inconsistent offsets, lengths or permutations come back as an error instead of reaching a kernel
(every bad case below is rejected on the host; nothing is launched for it)."""
import os

import numpy as np
import pytest

from paper_2608_27206_amd import workloads as wl
from tests.gpu_util import dev_bf16, dev_f32, dev_i32, say

pytestmark = pytest.mark.gpu


@pytest.fixture
def debug_env():
    old = os.environ.get("PACE_DEBUG")
    os.environ["PACE_DEBUG"] = "1"
    yield
    if old is None:
        del os.environ["PACE_DEBUG"]
    else:
        os.environ["PACE_DEBUG"] = old


def test_vit_attention_offsets(debug_env):
    from paper_2608_27206_amd import pace
    import torch
    N, H, d = 300, 2, 80
    q, k, v = (dev_bf16(wl.random_bf16(s, (N, H, d))) for s in (1, 2, 3))
    for cu, max_len, what in (([0, N + 5], N, "past the end"), ([0, 200, 150, N], N, "not monotone"),
                              ([0, 100, N], 150, "longer than max_seglen"), ([3, N], N, "not from 0")):
        say(f"bad cu_seqlens ({what})")
        with pytest.raises(pace.PaceError, match="cu_seqlens|offsets|segment"):
            pace.vit_attention(q, k, v, dev_i32(cu), max_len)
    # consistent offsets pass the check and run
    o, lse, mass = pace.vit_attention(q, k, v, dev_i32([0, 100, N]), 200)
    torch.cuda.synchronize()
    assert torch.isfinite(lse).all()


def test_prefill_metadata(debug_env):
    from paper_2608_27206_amd import pace
    L, Hq, Hkv, d = 96, 4, 2, 128
    q = dev_bf16(wl.random_bf16(4, (L, Hq, d)))
    k = dev_bf16(wl.random_bf16(5, (L, Hkv, d)))
    v = dev_bf16(wl.random_bf16(6, (L, Hkv, d)))
    cu = dev_i32([0, L])
    good = dict(vis=[64], cuv=[0, 64], ms=[64], ml=[32])
    bad_cases = [dict(good, vis=[100], cuv=[0, 100]),      # more visual tokens than the sequence
                 dict(good, cuv=[0, 60]),                   # cu_vis step differs from vis_len
                 dict(good, ms=[80], ml=[32])]              # querying rows past the end
    for c in bad_cases:
        say(f"bad prefill metadata {c}")
        with pytest.raises(pace.PaceError, match="pace_prefill_attention_with_mass"):
            pace.prefill_attention_with_mass(q, k, v, cu, L, dev_i32(c["vis"]), dev_i32(c["cuv"]),
                                             c["cuv"][-1], max(c["vis"]), dev_i32(c["ms"]), dev_i32(c["ml"]),
                                             max(c["ml"]))
    pace.prefill_attention_with_mass(q, k, v, cu, L, dev_i32(good["vis"]), dev_i32(good["cuv"]), 64, 64,
                                     dev_i32(good["ms"]), dev_i32(good["ml"]), 32)


def test_ddae_permutation(debug_env):
    from paper_2608_27206_amd import pace
    rs = np.random.default_rng(2)
    nvs = [40, 24]
    vis = dev_f32(rs.random((2, 4 * 64)))
    llm = dev_f32(rs.random((3, 64)))
    perm = np.concatenate([rs.permutation(40), rs.permutation(24)]).astype(np.int32)
    bad = perm.copy()
    bad[45] = 30   # image 1 has only 24 tokens
    say("bad vis_perm")
    with pytest.raises(pace.PaceError, match="vis_perm"):
        pace.ddae_select(vis, 4, dev_i32(bad), llm, nvs, [4, 3])
    pace.ddae_select(vis, 4, dev_i32(perm), llm, nvs, [4, 3])
