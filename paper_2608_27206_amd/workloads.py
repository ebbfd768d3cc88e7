"""Seeded synthetic inputs for the PACE hot path.

This module only draws random inputs and lays out token orders; it holds none of
the method's arithmetic (no density, attention, fusion or selection), so both
the HIP path and the CPU oracle can be fed from it without sharing any of the
computation under test.

Every array comes from ``numpy.random.default_rng([config_id, stream_id])``
(PCG64), so the same inputs appear on every machine.  Floating point tensors are
drawn in float32 and rounded to bfloat16 (round to nearest even); they are kept
as raw ``uint16`` bit patterns, which is what the device kernels consume.

Workload shapes follow Qwen2.5-VL-7B as used by the paper (Section 4.1, and the
complexity model of the appendix): 14-pixel patches, 2x2 spatial merge to the
LLM tokens, 8x8-patch window attention plus full attention in the vision
encoder (16 heads, head dim 80) and grouped-query prefill attention in the LLM
(28 query heads, 4 KV heads, head dim 128, hidden size 3584).
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import Dict, List, Optional

import numpy as np

PATCH = 14
MERGE = 2          # 2x2 spatial merge: 4 patches -> 1 LLM visual token
WINDOW = 8         # window attention over 8x8 patches
VIT_HEADS = 16
VIT_DIM = 80
LLM_QHEADS = 28
LLM_KVHEADS = 4
LLM_DIM = 128
HIDDEN = 3584

# stream ids of the seeded generators
S_Q, S_K, S_V, S_SAL_PICK, S_SAL_DIR, S_VITMASS, S_HIDDEN, S_IMAGE, S_RES, S_TEXT = range(10)

CONFIG_NAMES = {
    0: "tiny_prefill_196v_32t",
    1: "img448_qwen25vl7b",
    2: "img1344_qwen25vl7b",
    3: "frame4k_3836x2156_qwen25vl7b",
    4: "varlen8_qwen25vl7b",
}


def rng(config_id: int, stream: int) -> np.random.Generator:
    return np.random.default_rng([int(config_id), int(stream)])


# ---------------------------------------------------------------- bf16 helpers
def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round float32 to bfloat16 (nearest even) and return the uint16 bit patterns."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    bias = ((u >> 16) & 1) + 0x7FFF
    return ((u + bias) >> 16).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << 16).view(np.float32)


def bf16_bits_to_f64(b: np.ndarray) -> np.ndarray:
    return bf16_bits_to_f32(b).astype(np.float64)


# ---------------------------------------------------------------- images
def make_image(config_id: int, H: int, W: int, stream: int = S_IMAGE,
               textured_frac: float = 0.20, level: float = 127.5, amplitude: float = 100.0) -> np.ndarray:
    """uint8 HWC RGB image: smooth per-channel sinusoids around `level` with the given
    amplitude, with a seeded fraction of the 14x14 patches replaced by uniform random
    texture."""
    g = rng(config_id, stream)
    a = g.uniform(0.5, 2.0, size=3)
    b = g.uniform(0.5, 2.0, size=3)
    ph = g.uniform(0.0, 2.0 * math.pi, size=3)
    y = np.arange(H, dtype=np.float64)[:, None]
    x = np.arange(W, dtype=np.float64)[None, :]
    img = np.empty((H, W, 3), dtype=np.uint8)
    for c in range(3):
        v = level + amplitude * np.sin(2.0 * math.pi * (a[c] * x / W + b[c] * y / H) + ph[c])
        img[:, :, c] = np.clip(np.floor(v + 0.5), 0, 255).astype(np.uint8)
    gh, gw = H // PATCH, W // PATCH
    n = gh * gw
    if n > 0 and textured_frac > 0:
        ntex = int(math.ceil(textured_frac * n))
        pick = g.choice(n, size=ntex, replace=False)
        tex = g.integers(0, 256, size=(ntex, PATCH, PATCH, 3), dtype=np.uint8)
        for t, p in enumerate(pick):
            py, px = divmod(int(p), gw)
            img[py * PATCH:(py + 1) * PATCH, px * PATCH:(px + 1) * PATCH, :] = tex[t]
    return img


def varlen_image_styles(config_id: int = 4, count: int = 8):
    """Seeded per-image (level, amplitude, textured fraction): from document-like pages (bright,
    flat, sparse detail) to busy scenes, so APC's density differs between images."""
    g = rng(config_id, S_IMAGE)
    return [(float(g.uniform(60.0, 235.0)), float(g.uniform(3.0, 80.0)), float(g.uniform(0.01, 0.30)))
            for _ in range(count)]


# ---------------------------------------------------------------- token layout
@dataclass
class VitLayout:
    gh: int                      # patch rows
    gw: int                      # patch columns
    order: np.ndarray            # [N] raster patch index of each ViT token (window-major)
    cu_windows: np.ndarray       # [nwin+1] int32 window boundaries in ViT token order
    vis_perm: np.ndarray         # [N/4] int32: LLM raster token i -> merged ViT token index
    window_sizes: List[int] = field(default_factory=list)

    @property
    def n_patches(self) -> int:
        return self.gh * self.gw

    @property
    def n_vis(self) -> int:
        return (self.gh // MERGE) * (self.gw // MERGE)


def vit_layout(gh: int, gw: int, window: int = WINDOW, merge: int = MERGE) -> VitLayout:
    """Window-major token order of a Qwen2.5-VL style encoder.

    Windows of ``window x window`` patches in raster order; inside a window the
    ``merge x merge`` groups in raster order; inside a group its patches in raster
    order.  Partial windows at the right and bottom edges hold what is left.
    Requires gh and gw to be multiples of ``merge``."""
    assert gh % merge == 0 and gw % merge == 0 and window % merge == 0
    mh, mw = gh // merge, gw // merge
    wm = window // merge
    order = []
    cu = [0]
    merged_index = np.full((mh, mw), -1, dtype=np.int64)
    m_counter = 0
    sizes = []
    for wy in range(0, mh, wm):
        for wx in range(0, mw, wm):
            start = len(order)
            for my in range(wy, min(wy + wm, mh)):
                for mx in range(wx, min(wx + wm, mw)):
                    merged_index[my, mx] = m_counter
                    m_counter += 1
                    for dy in range(merge):
                        for dx in range(merge):
                            py, px = my * merge + dy, mx * merge + dx
                            order.append(py * gw + px)
            cu.append(len(order))
            sizes.append(len(order) - start)
    vis_perm = merged_index.reshape(-1).astype(np.int32)
    return VitLayout(gh=gh, gw=gw, order=np.asarray(order, dtype=np.int64),
                     cu_windows=np.asarray(cu, dtype=np.int32), vis_perm=vis_perm,
                     window_sizes=sizes)


# ---------------------------------------------------------------- workloads
@dataclass
class PrefillInputs:
    q: np.ndarray                # bf16 bits [Ntot, Hq, d]
    k: np.ndarray                # bf16 bits [Ntot, Hkv, d]
    v: np.ndarray                # bf16 bits [Ntot, Hkv, d]
    cu_seqlens: np.ndarray       # int32 [B+1]
    vis_len: np.ndarray          # int32 [B]   visual tokens lead each sequence
    text_len: np.ndarray         # int32 [B]
    cu_vis: np.ndarray           # int32 [B+1] offsets of each sequence's visual keys in mass
    salient: List[np.ndarray]    # per sequence: visual token ids made salient
    q_f32: Optional[np.ndarray] = None   # tiny config: pre-rounding float32 values of q, k, v
    k_f32: Optional[np.ndarray] = None
    v_f32: Optional[np.ndarray] = None

    @property
    def mq_start(self) -> np.ndarray:
        """Mass is read from the text rows, which follow the visual rows."""
        return self.vis_len.astype(np.int32)

    @property
    def mq_len(self) -> np.ndarray:
        return self.text_len.astype(np.int32)


@dataclass
class VitInputs:
    q: np.ndarray                # bf16 bits [N, H, d], window-major token order
    k: np.ndarray
    v: np.ndarray
    cu_full: np.ndarray          # int32 [B+1]: one segment per image
    cu_windows: np.ndarray       # int32 [nwin+1]
    vis_perm: np.ndarray         # int32 [sum N_vis]: per image, LLM raster -> merged ViT order
    cu_vis: np.ndarray           # int32 [B+1] merged-token offsets per image


@dataclass
class Workload:
    config_id: int
    name: str
    images: List[np.ndarray]               # uint8 HWC, one per image (may be empty)
    layouts: List[VitLayout]
    vit: Optional[VitInputs]
    prefill: PrefillInputs
    vit_mass: Optional[np.ndarray]         # fp32 [Hv, Nv*merge] given directly (tiny config)
    vit_merge: int
    hidden: np.ndarray                     # bf16 bits [sum N_vis, HIDDEN]
    keep_ratio: float                      # fixed ratio (per-image ratios come from APC in varlen)
    fusion_mode: int                       # 0 dynamic softmax(sigma/tau), 1 fixed weights
    tau: float = 0.5
    w_llm_fixed: float = 0.5
    downsample_scale: Optional[float] = None   # fixed resize factor per side (4K frame)
    meta: Dict = field(default_factory=dict)


def _normal_bf16(config_id: int, stream: int, shape, scale: float = 1.0):
    g = rng(config_id, stream)
    x = g.standard_normal(size=shape, dtype=np.float32)
    if scale != 1.0:
        x *= np.float32(scale)
    return x


def _prefill(config_id: int, vis_lens: List[int], text_lens: List[int], hq: int, hkv: int,
             d: int, qkv_scale: float, salient: bool, keep_f32: bool = False) -> PrefillInputs:
    seqlens = [a + b for a, b in zip(vis_lens, text_lens)]
    ntot = int(sum(seqlens))
    q = _normal_bf16(config_id, S_Q, (ntot, hq, d), qkv_scale)
    k = _normal_bf16(config_id, S_K, (ntot, hkv, d), qkv_scale)
    v = _normal_bf16(config_id, S_V, (ntot, hkv, d), qkv_scale)
    sal_list = []
    if salient:
        gp = rng(config_id, S_SAL_PICK)
        gd = rng(config_id, S_SAL_DIR)
        u = gd.standard_normal(size=(hkv, d))
        u /= np.linalg.norm(u, axis=1, keepdims=True)
        off = 0
        for nv, s in zip(vis_lens, seqlens):
            nsal = int(math.ceil(0.05 * nv))
            pick = np.sort(gp.choice(nv, size=nsal, replace=False))
            k[off + pick, :, :] += (3.0 * u)[None, :, :].astype(np.float32)
            sal_list.append(pick.astype(np.int64))
            off += s
    cu = np.zeros(len(seqlens) + 1, dtype=np.int32)
    cu[1:] = np.cumsum(seqlens)
    cuv = np.zeros(len(vis_lens) + 1, dtype=np.int32)
    cuv[1:] = np.cumsum(vis_lens)
    return PrefillInputs(
        q=f32_to_bf16_bits(q), k=f32_to_bf16_bits(k), v=f32_to_bf16_bits(v),
        cu_seqlens=cu, vis_len=np.asarray(vis_lens, dtype=np.int32),
        text_len=np.asarray(text_lens, dtype=np.int32), cu_vis=cuv, salient=sal_list,
        q_f32=(q if keep_f32 else None), k_f32=(k if keep_f32 else None), v_f32=(v if keep_f32 else None))


def _vit(config_id: int, layouts: List[VitLayout]) -> VitInputs:
    n = sum(L.n_patches for L in layouts)
    q = f32_to_bf16_bits(_normal_bf16(config_id, S_Q + 100, (n, VIT_HEADS, VIT_DIM)))
    k = f32_to_bf16_bits(_normal_bf16(config_id, S_K + 100, (n, VIT_HEADS, VIT_DIM)))
    v = f32_to_bf16_bits(_normal_bf16(config_id, S_V + 100, (n, VIT_HEADS, VIT_DIM)))
    cu_full = [0]
    cu_win = [0]
    perms = []
    cu_vis = [0]
    for L in layouts:
        base = cu_full[-1]
        cu_win.extend((base + L.cu_windows[1:]).tolist())
        cu_full.append(base + L.n_patches)
        perms.append(L.vis_perm)
        cu_vis.append(cu_vis[-1] + L.n_vis)
    return VitInputs(q=q, k=k, v=v, cu_full=np.asarray(cu_full, dtype=np.int32),
                     cu_windows=np.asarray(cu_win, dtype=np.int32),
                     vis_perm=np.concatenate(perms).astype(np.int32),
                     cu_vis=np.asarray(cu_vis, dtype=np.int32))


def random_bf16(seed: int, shape, scale: float = 1.0) -> np.ndarray:
    """bf16 bits of N(0, scale^2) draws from rng([1000 + seed, 0]) (test shapes)."""
    return f32_to_bf16_bits(_normal_bf16(1000 + seed, 0, shape, scale))


def preview_weights(seed: int, dim: int = 1280, ffn: int = 3420, patch: int = 14) -> dict:
    """Seeded weights of a vision-encoder block of Qwen2.5-VL-7B's shapes (the APC preview):
    bf16 bit arrays for the matrices (N(0,1)/sqrt(fan_in)), fp32 for biases (N(0, 0.02)) and
    RMSNorm gains (1 + N(0, 0.1)).  Only random numbers, no arithmetic of the method."""
    g = np.random.default_rng([seed, 77])
    kin = 3 * patch * patch

    def mat(n, k):
        return f32_to_bf16_bits((g.standard_normal((n, k)) / np.sqrt(k)).astype(np.float32))

    def vec(n, scale):
        return (g.standard_normal(n) * scale).astype(np.float32)

    w = {"pe": mat(dim, kin), "g1": (1.0 + vec(dim, 0.1)).astype(np.float32)}
    for name in ("q", "k", "v", "o"):
        w["w" + name] = mat(dim, dim)
        w["b" + name] = vec(dim, 0.02)
    w["g2"] = (1.0 + vec(dim, 0.1)).astype(np.float32)
    w["wg"], w["bg"] = mat(ffn, dim), vec(ffn, 0.02)
    w["wu"], w["bu"] = mat(ffn, dim), vec(ffn, 0.02)
    w["wd"], w["bd"] = mat(dim, ffn), vec(dim, 0.02)
    return w


def _hidden(config_id: int, nv: int) -> np.ndarray:
    return f32_to_bf16_bits(_normal_bf16(config_id, S_HIDDEN, (nv, HIDDEN)))


def varlen_resolutions(config_id: int = 4, count: int = 8):
    """Seeded (H, W) pairs, multiples of 28, between 448x448 and 2240x1260 (W x H)."""
    g = rng(config_id, S_RES)
    ws = g.integers(448 // 28, 2240 // 28 + 1, size=count) * 28
    hs = g.integers(448 // 28, 1260 // 28 + 1, size=count) * 28
    return [(int(h), int(w)) for h, w in zip(hs, ws)]


def make_workload(config_id: int) -> Workload:
    name = CONFIG_NAMES[config_id]
    if config_id == 0:
        nv, nt = 196, 32
        pre = _prefill(0, [nv], [nt], 8, 2, 128, 1.0 / math.sqrt(128.0), salient=True,
                       keep_f32=True)
        vm = rng(0, S_VITMASS).dirichlet(np.ones(nv)).astype(np.float32)[None, :]
        return Workload(config_id=0, name=name, images=[], layouts=[], vit=None, prefill=pre,
                        vit_mass=vm, vit_merge=1, hidden=_hidden(0, nv), keep_ratio=0.10,
                        fusion_mode=1, w_llm_fixed=0.5)
    if config_id in (1, 2, 3):
        H, W = {1: (448, 448), 2: (1344, 1344), 3: (2156, 3836)}[config_id]
        text = {1: 64, 2: 128, 3: 128}[config_id]
        img = make_image(config_id, H, W)
        L = vit_layout(H // PATCH, W // PATCH)
        vit = _vit(config_id, [L])
        pre = _prefill(config_id, [L.n_vis], [text], LLM_QHEADS, LLM_KVHEADS, LLM_DIM, 1.0,
                       salient=(config_id != 1))
        return Workload(config_id=config_id, name=name, images=[img], layouts=[L], vit=vit,
                        prefill=pre, vit_mass=None, vit_merge=MERGE,
                        hidden=_hidden(config_id, L.n_vis), keep_ratio=0.10, fusion_mode=0,
                        downsample_scale=(0.5 if config_id == 3 else None))
    if config_id == 4:
        res = varlen_resolutions(4)
        styles = varlen_image_styles(4, len(res))
        imgs = [make_image(4, h, w, stream=S_IMAGE * 100 + i, textured_frac=tf, level=lv, amplitude=am)
                for i, ((h, w), (lv, am, tf)) in enumerate(zip(res, styles))]
        lays = [vit_layout(h // PATCH, w // PATCH) for (h, w) in res]
        vit = _vit(4, lays)
        gt = rng(4, S_TEXT)
        texts = [int(t) for t in gt.integers(64, 257, size=len(res))]
        pre = _prefill(4, [L.n_vis for L in lays], texts, LLM_QHEADS, LLM_KVHEADS, LLM_DIM, 1.0,
                       salient=True)
        nv = sum(L.n_vis for L in lays)
        return Workload(config_id=4, name=name, images=imgs, layouts=lays, vit=vit, prefill=pre,
                        vit_mass=None, vit_merge=MERGE, hidden=_hidden(4, nv), keep_ratio=0.10,
                        fusion_mode=0, meta={"resolutions": res, "text_lens": texts, "styles": styles})
    raise ValueError(f"unknown config {config_id}")
