"""The first extensions beyond the hot path, at the same parity bar.

- Compaction after pruning: the kept indices DDAE produced gather every per-token tensor
  of the shortened context (Q/K/V rows, position ids) bit for bit, and the same prefill
  kernel then runs on the T + K remaining tokens (Section 3.3: the kept tokens form the
  LLM's shortened context).  Checked against the oracle on the same compacted inputs.
- The all-query ("Vision + Text") source of S_llm is the prefill mass with every row of
  the sequence querying (covered by test_prefill_all_rows_mass); here at the 1344^2 shapes."""
import math

import numpy as np
import pytest

from oracle import attention as oatt
from oracle import ddae as oddae
from paper_2608_27206_amd import workloads as wl
from tests.gpu_util import dev_bf16, dev_f32, dev_i32, host, host_bf16_to_f64, mass_ok, say

pytestmark = pytest.mark.gpu

O_TOL, LSE_TOL = 2e-2, 1e-3


def test_gather_rows_bit_exact_and_skips_out_of_range():
    from paper_2608_27206_amd import pace
    import torch
    rs = np.random.default_rng(3)
    src = wl.random_bf16(3, (500, 3584))
    idx = rs.integers(0, 500, 300).astype(np.int32)
    idx[[7, 100]] = [-1, 500]          # out of range: the rows stay as they were
    out = torch.full((300, 3584), 7.0, dtype=torch.bfloat16, device="cuda")
    pace.gather_rows(dev_bf16(src), dev_i32(idx), out=out)
    torch.cuda.synchronize()
    got = out.view(torch.int16).cpu().numpy().view(np.uint16)
    ok = (idx >= 0) & (idx < 500)
    np.testing.assert_array_equal(got[ok], src[idx[ok]])
    seven = np.uint16(0x40E0)          # bf16 bits of 7.0
    assert np.all(got[~ok] == seven)
    pos = rs.integers(0, 1 << 20, (500, 4)).astype(np.int32)   # position ids padded to 16 B
    gp = pace.gather_rows(dev_i32(pos), dev_i32(np.where(ok, idx, 0)))
    np.testing.assert_array_equal(host(gp), pos[np.where(ok, idx, 0)])


def test_post_prune_prefill_chain():
    """Prefill with text-query mass -> DDAE select (10%) -> gather Q/K/V/positions of the
    kept visual tokens and all text tokens -> prefill on the shortened sequence."""
    from paper_2608_27206_amd import pace
    import torch
    w = wl.make_workload(2)
    p = w.prefill
    nv, T = int(p.vis_len[0]), int(p.text_len[0])
    S = nv + T
    say(f"post-prune chain: {nv} visual + {T} text tokens")
    Q, Kt, V = dev_bf16(p.q), dev_bf16(p.k), dev_bf16(p.v)
    _, _, mass_llm = pace.prefill_attention_with_mass(
        Q, Kt, V, dev_i32(p.cu_seqlens), S, dev_i32(p.vis_len), dev_i32(p.cu_vis), nv, nv,
        dev_i32(p.mq_start), dev_i32(p.mq_len), T)
    rs = np.random.default_rng(11)
    vis = rs.gamma(0.5, size=(16, 4 * nv)).astype(np.float32)
    K = oddae.keep_count(0.10, nv)
    idx, scores, _, _ = pace.ddae_select(dev_f32(vis), 4, dev_i32(w.vit.vis_perm), mass_llm, [nv], [K])
    keep = torch.cat([idx.long(), torch.arange(nv, S, device="cuda")]).to(torch.int32)
    Sp = K + T
    Qc = pace.gather_rows(Q, keep)
    Kc = pace.gather_rows(Kt, keep)
    Vc = pace.gather_rows(V, keep)
    pos = np.stack([np.arange(S), np.arange(S) // 7, np.arange(S) % 11, np.zeros(S)], 1).astype(np.int32)
    posc = pace.gather_rows(dev_i32(pos), keep)
    cu = dev_i32([0, Sp])
    o, lse, mass = pace.prefill_attention_with_mass(
        Qc, Kc, Vc, cu, Sp, dev_i32([K]), dev_i32([0, K]), K, K, dev_i32([K]), dev_i32([T]), T)
    torch.cuda.synchronize()
    keep_h = host(keep).astype(np.int64)
    # the kept set is the selection's (ascending visual indices, then the text tokens)
    assert np.all(np.diff(keep_h[:K]) > 0) and keep_h[K - 1] < nv
    np.testing.assert_array_equal(keep_h[:K], oddae.topk_indices(host(scores), K))
    np.testing.assert_array_equal(host(posc), pos[keep_h])
    for name, dev_t, src in (("q", Qc, p.q), ("k", Kc, p.k), ("v", Vc, p.v)):
        got = dev_t.view(torch.int16).cpu().numpy().view(np.uint16)
        np.testing.assert_array_equal(got, src[keep_h], err_msg=name)
    # prefill on the compacted sequence against the oracle on the same compacted inputs
    qc, kc, vc = (wl.bf16_bits_to_f64(a[keep_h]) for a in (p.q, p.k, p.v))
    o_h, lse_h, mass_h = host_bf16_to_f64(o), host(lse), host(mass)
    rows = np.unique(np.concatenate([[0, K - 1, K, Sp - 1], rs.integers(0, Sp, 12)]))
    hq, hkv = p.q.shape[1], p.k.shape[1]
    scale = 1 / math.sqrt(p.q.shape[2])
    for h in range(hq):
        kv = h // (hq // hkv)
        O, L, M = oatt.attention_segment(qc[:, h:h + 1], kc[:, kv:kv + 1], vc[:, kv:kv + 1], True,
                                         scale, rows=rows, mass_rows=np.arange(K, Sp))
        assert np.max(np.abs(o_h[rows, h] - O[:, 0])) <= O_TOL
        assert np.max(np.abs(lse_h[h, rows] - L[0])) <= LSE_TOL
        err, rel = mass_ok(mass_h[h, :K], M[0, :K], T)
        assert err <= 0, (h, rel)
