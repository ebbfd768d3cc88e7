"""The seeded generators: shapes of the paper's Qwen2.5-VL-7B workloads and determinism."""
import numpy as np
import pytest

from paper_2608_27206_amd import workloads as wl


def test_bf16_round_trip_and_rne():
    x = np.array([1.0, -2.5, 3.1415926, 1e-3, 65504.0], np.float32)
    b = wl.f32_to_bf16_bits(x)
    y = wl.bf16_bits_to_f32(b)
    assert np.all(np.abs(y - x) <= np.abs(x) * 2 ** -8)
    # ties to even: 1 + 2^-8 is halfway between 1 and 1 + 2^-7 -> rounds to 1
    t = np.array([1 + 2 ** -8, 1 + 3 * 2 ** -8], np.float32)
    np.testing.assert_array_equal(wl.bf16_bits_to_f32(wl.f32_to_bf16_bits(t)), [1.0, 1 + 2 ** -6])


def test_4k_window_layout():
    L = wl.vit_layout(154, 274)
    assert L.n_patches == 42196 and L.n_vis == 10549
    sizes = np.diff(L.cu_windows)
    assert len(sizes) == 700
    assert (sizes == 64).sum() == 646 and (sizes == 16).sum() == 53 and (sizes == 4).sum() == 1
    assert sorted(L.order.tolist()) == list(range(42196))
    assert sorted(L.vis_perm.tolist()) == list(range(10549))


def test_window_order_groups_merge_quads():
    L = wl.vit_layout(4, 6, window=4)
    # first merged group of the first window: patches (0,0), (0,1), (1,0), (1,1)
    assert L.order[:4].tolist() == [0, 1, 6, 7]
    # LLM raster token (0, 2) (third merged column) sits in the second window
    assert L.vis_perm[2] == 4


def test_tiny_config_shapes_and_determinism():
    a = wl.make_workload(0)
    b = wl.make_workload(0)
    p = a.prefill
    assert p.q.shape == (228, 8, 128) and p.k.shape == (228, 2, 128)
    assert p.vis_len.tolist() == [196] and p.text_len.tolist() == [32]
    assert len(p.salient[0]) == 10
    assert a.vit_mass.shape == (1, 196) and abs(float(a.vit_mass.sum()) - 1) < 1e-5
    assert a.hidden.shape == (196, 3584)
    np.testing.assert_array_equal(a.prefill.k, b.prefill.k)
    np.testing.assert_array_equal(a.hidden, b.hidden)


def test_img448_shapes():
    w = wl.make_workload(1)
    assert w.images[0].shape == (448, 448, 3) and w.images[0].dtype == np.uint8
    assert w.vit.q.shape == (1024, 16, 80)
    assert w.vit.cu_windows.tolist() == list(range(0, 1025, 64))
    assert w.prefill.q.shape == (320, 28, 128)


def test_varlen_resolutions_in_range():
    res = wl.varlen_resolutions()
    assert len(res) == 8
    for h, w in res:
        assert 448 <= h <= 1260 and 448 <= w <= 2240 and h % 28 == 0 and w % 28 == 0
