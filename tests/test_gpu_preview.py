"""GPU parity of the APC preview block (pace_apc_preview, pace_gemm_bf16) against the float64
oracle (oracle/preview.py).

GEMM: every output within 2^-8 of |ref| (its bf16 rounding) plus 1e-3 of the output's RMS
(fp32 accumulation over K).  Block: the GPU stores ten intermediate activations in bf16
(relative rounding 2^-9 each), and each passes through products of depth up to 3420. Summed over
the chain that is about 2% for a single worst element and well under 1% in RMS. So the output's
RMS error is bounded by 1e-2 of the output RMS and its largest error by 6e-2 of it, and every
row's cosine with the oracle's must be >= 0.999. The APC scores computed from the GPU embeddings
agree with the oracle's scores of the oracle embeddings to 2e-3."""
import numpy as np
import pytest

from oracle import apc as oapc
from oracle import preview as opv
from paper_2608_27206_amd import workloads as wl
from tests.gpu_util import dev_bf16, dev_f32, dev_i32, dev_u8, host, host_bf16_to_f64, rho4, say

pytestmark = pytest.mark.gpu


def _silu(x):
    return x / (1.0 + np.exp(-x))


@pytest.mark.parametrize("M,N,K,epi", [(300, 200, 72, 0), (1024, 1280, 1280, 0), (129, 257, 8, 1),
                                       (513, 384, 592, 1), (200, 96, 1280, 2), (1, 2, 16, 2)])
def test_gemm_epilogues(M, N, K, epi):
    from paper_2608_27206_amd import pace
    import torch
    say(f"gemm M={M} N={N} K={K} epilogue={epi}")
    rs = np.random.default_rng(M * 7 + N + K)
    a = wl.f32_to_bf16_bits(rs.normal(size=(M, K)).astype(np.float32))
    b = wl.f32_to_bf16_bits((rs.normal(size=(N, K)) / np.sqrt(K)).astype(np.float32))
    bias = rs.normal(size=N).astype(np.float32) * 0.1
    res = wl.f32_to_bf16_bits(rs.normal(size=(M, N)).astype(np.float32))
    out = pace.gemm_bf16(dev_bf16(a), dev_bf16(b), dev_f32(bias), dev_bf16(res) if epi == 1 else None, epi)
    torch.cuda.synchronize()
    got = host_bf16_to_f64(out)
    ref = wl.bf16_bits_to_f64(a) @ wl.bf16_bits_to_f64(b).T + bias[None, :]
    if epi == 1:
        ref = ref + wl.bf16_bits_to_f64(res)
    if epi == 2:
        ref = _silu(ref[:, 0::2]) * ref[:, 1::2]
    tol = 2.0 ** -8 * np.abs(ref) + 1e-3 * np.sqrt(np.mean(ref ** 2))
    assert np.all(np.abs(got - ref) <= tol), float(np.max(np.abs(got - ref) - tol))


def _block_case(H, W, seed=11):
    from paper_2608_27206_amd import pace
    import torch
    img = wl.make_image(1, H, W)
    lay = wl.vit_layout(H // 14, W // 14)
    w = wl.preview_weights(seed)
    wdev = pace.preview_weights_to_device(w, torch.device("cuda"))
    out = pace.apc_preview(dev_u8(img), 14, dev_i32(lay.order), dev_i32(lay.cu_windows),
                           int(np.max(lay.window_sizes)), wdev)
    rho, d = pace.apc_density_features(out)
    torch.cuda.synchronize()
    w64 = {k: (wl.bf16_bits_to_f64(v) if v.dtype == np.uint16 else v.astype(np.float64)) for k, v in w.items()}
    ref = opv.preview_block(opv.patch_rows(img, 14, lay.order), w64, lay.cu_windows)
    return host_bf16_to_f64(out), ref, host(rho), host(d)


def _check_block(got, ref, name):
    rms = np.sqrt(np.mean(ref ** 2))
    err = got - ref
    rel_max = np.max(np.abs(err)) / rms
    rel_rms = np.sqrt(np.mean(err ** 2)) / rms
    cos = np.sum(got * ref, axis=1) / (np.linalg.norm(got, axis=1) * np.linalg.norm(ref, axis=1))
    say(f"preview {name}: max err / rms = {rel_max:.3g}, rms err / rms = {rel_rms:.3g}, "
        f"min row cosine = {cos.min():.6f}")
    assert rel_rms <= 1e-2
    assert rel_max <= 6e-2
    assert cos.min() >= 0.999


def test_preview_block_448():
    got, ref, rho, d = _block_case(448, 448)
    _check_block(got, ref, "448")
    dens = oapc.embedding_density(ref)
    say(f"rho gpu {rho} oracle {[dens['rho_g'], dens['rho_d'], dens['rho'], dens['phi']]}")
    np.testing.assert_allclose(rho4(rho), [dens["rho_g"], dens["rho_d"], dens["rho"], dens["phi"]], atol=2e-3)


def test_preview_block_ragged_windows():
    """A grid whose windows are cut at the right and bottom edges (partial windows)."""
    got, ref, rho, d = _block_case(196, 308, seed=12)
    _check_block(got, ref, "196x308")
