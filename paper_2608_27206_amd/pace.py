"""ctypes binding of libpace.so (include/pace.h): argument marshalling only.

Every function takes torch tensors that already live on the GPU, passes their
device pointers and torch's current HIP stream to the C ABI, and returns the
output tensors it allocated with torch.  All arithmetic happens in the HIP
kernels; if the library is missing this module raises instead of computing
anything itself.
"""
from __future__ import annotations

import ctypes
import math
import os
from typing import Optional, Sequence

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
# PACE_LIB_PATH selects another build of the same library (the host-sanitized one of the C ABI
# tests); by default the in-tree libpace.so.
LIB_PATH = os.environ.get("PACE_LIB_PATH") or os.path.join(_HERE, "libpace.so")

_lib = None

c_int, c_size, c_double, c_float, c_void = (ctypes.c_int, ctypes.c_size_t, ctypes.c_double,
                                            ctypes.c_float, ctypes.c_void_p)
c_int_p = ctypes.POINTER(ctypes.c_int)

# name -> (restype, argtypes)
_PROTOS = {
    "pace_last_error": (ctypes.c_char_p, []),
    "pace_version": (c_int, []),
    "pace_keep_count": (c_int, [c_double, c_int]),
    "pace_keep_from_density": (c_int, [c_double, c_double, c_double, c_int]),
    "pace_apc_target_size": (c_int, [c_double, c_int, c_int, c_double, c_double, c_int, c_int_p,
                                     c_int_p]),
    "pace_apc_density_workspace_size": (c_size, [c_int, c_int, c_int]),
    "pace_apc_density": (c_int, [c_void, c_int, c_int, c_int, c_double, c_float, c_float, c_void,
                                 c_void, c_void, c_size, c_void]),
    "pace_apc_density_features_workspace_size": (c_size, [c_int, c_int]),
    "pace_apc_density_features": (c_int, [c_void, c_int, c_int, c_double, c_float, c_float, c_void,
                                          c_void, c_void, c_size, c_void]),
    "pace_apc_downsample": (c_int, [c_void, c_int, c_int, c_void, c_int, c_int, c_void]),
    "pace_apc_pixel_features": (c_int, [c_void, c_int, c_int, c_int, c_int, c_void, c_void]),
    "pace_apc_pixel_density_workspace_size": (c_size, [c_int, c_int, c_int, c_int]),
    "pace_apc_pixel_density": (c_int, [c_void, c_int, c_int, c_int, c_int, c_double, c_float, c_float,
                                       c_void, c_void, c_void, c_size, c_void]),
    "pace_apc_preview_workspace_size": (c_size, [c_int, c_int, c_int, c_int]),
    "pace_apc_preview": (c_int, [c_void, c_int, c_int, c_int, c_void, c_void, c_int, c_int, c_void, c_void,
                                 c_void, c_size, c_void]),
    "pace_gemm_bf16": (c_int, [c_void, c_void, c_void, c_void, c_void, c_int, c_int, c_int, c_int, c_void]),
    "pace_vit_attention_workspace_size": (c_size, [c_int, c_int, c_int, c_int, c_int]),
    "pace_vit_attention": (c_int, [c_void, c_void, c_void, c_int, c_int, c_int, c_void, c_int, c_int,
                                   c_float, c_void, c_void, c_void, c_void, c_size, c_void]),
    "pace_vit_attention_mass": (c_int, [c_void, c_void, c_int, c_int, c_int, c_void, c_int, c_int,
                                        c_float, c_void, c_void, c_void]),
    "pace_prefill_attention_workspace_size": (c_size, [c_int, c_int]),
    "pace_prefill_attention_with_mass": (c_int, [c_void, c_void, c_void, c_int, c_int, c_int, c_int,
                                                 c_void, c_int, c_int, c_void, c_void, c_void, c_int, c_int,
                                                 c_void, c_void, c_int, c_float, c_void, c_void,
                                                 c_void, c_void, c_size, c_void]),
    "pace_ddae_select_workspace_size": (c_size, [c_int, c_int]),
    "pace_ddae_select_varlen": (c_int, [c_void, c_int, c_int, c_void, c_void, c_int, c_int, c_int_p,
                                        c_int_p, c_int, c_float, c_float, c_void, c_size, c_void,
                                        c_void, c_void, c_void, c_void, c_size, c_void]),
    "pace_ddae_select": (c_int, [c_void, c_int, c_int, c_void, c_void, c_int, c_int, c_int, c_float,
                                 c_float, c_int, c_void, c_size, c_void, c_void, c_void, c_void,
                                 c_void, c_size, c_void]),
    "pace_ddae_select_noalloc_max_bytes": (c_size, []),
    "pace_ddae_select_varlen_noalloc": (c_int, [c_void, c_int, c_int, c_void, c_void, c_int, c_int, c_int_p,
                                                c_int_p, c_int, c_float, c_float, c_void, c_size, c_void,
                                                c_void, c_void, c_void, c_void]),
    "pace_topk_gather": (c_int, [c_void, c_int, c_int, c_void, c_size, c_void, c_void, c_void, c_size,
                                 c_void]),
    "pace_gather_rows": (c_int, [c_void, c_int, c_size, c_void, c_int, c_void, c_void]),
}

EXPORTED = tuple(_PROTOS.keys())


class PaceError(RuntimeError):
    pass


def lib():
    """Load libpace.so (built by paper_2608_27206_amd.build); raise if it is missing."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise PaceError(f"{LIB_PATH} is missing: run `python -m paper_2608_27206_amd.build`")
        L = ctypes.CDLL(LIB_PATH)
        for name, (res, args) in _PROTOS.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _lib = L
    return _lib


def _check(st: int, what: str):
    if st != 0:
        msg = lib().pace_last_error().decode(errors="replace")
        raise PaceError(f"{what} failed with status {st}: {msg}")


def _ptr(t: Optional[torch.Tensor]):
    if t is None:
        return None
    if not t.is_cuda:
        raise PaceError("tensor must live on the GPU")
    if not t.is_contiguous():
        raise PaceError("tensor must be contiguous")
    return ctypes.c_void_p(t.data_ptr())


def _stream():
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def _ws(nbytes: int, device) -> torch.Tensor:
    return torch.empty(max(1, int(nbytes)), dtype=torch.uint8, device=device)


# ---------------------------------------------------------------- host helpers
def keep_count(ratio: float, n: int) -> int:
    return int(lib().pace_keep_count(float(ratio), int(n)))


def keep_from_density(rho: float, n: int, ratio_lo: float = 0.05, ratio_hi: float = 0.25) -> int:
    return int(lib().pace_keep_from_density(float(rho), float(ratio_lo), float(ratio_hi), int(n)))


def apc_target_size(rho: float, H: int, W: int, min_pixels: float, max_pixels: float, snap: int):
    oh, ow = ctypes.c_int(0), ctypes.c_int(0)
    _check(lib().pace_apc_target_size(float(rho), H, W, float(min_pixels), float(max_pixels), snap,
                                      ctypes.byref(oh), ctypes.byref(ow)), "pace_apc_target_size")
    return oh.value, ow.value


# ---------------------------------------------------------------- APC
def apc_density(img: torch.Tensor, patch: int = 14, tail_frac: float = 0.10, alpha: float = 0.6,
                gamma: float = 1.5, d_out: Optional[torch.Tensor] = None,
                rho_out: Optional[torch.Tensor] = None, workspace: Optional[torch.Tensor] = None):
    """img: uint8 [H, W, 3] on the GPU.  Returns (rho [3] = rho_g, rho_d, rho; d [N]); phi = 1 - rho_g."""
    H, W, _ = img.shape
    N = (H // patch) * (W // patch)
    dev = img.device
    if d_out is None:
        d_out = torch.empty(N, dtype=torch.float32, device=dev)
    if rho_out is None:
        rho_out = torch.empty(3, dtype=torch.float32, device=dev)
    need = lib().pace_apc_density_workspace_size(H, W, patch)
    if workspace is None:
        workspace = _ws(need, dev)
    _check(lib().pace_apc_density(_ptr(img), H, W, patch, float(tail_frac), float(alpha),
                                  float(gamma), _ptr(d_out), _ptr(rho_out), _ptr(workspace),
                                  workspace.numel(), _stream()), "pace_apc_density")
    return rho_out, d_out


def apc_density_features(feat: torch.Tensor, tail_frac: float = 0.10, alpha: float = 0.6,
                         gamma: float = 1.5, d_out: Optional[torch.Tensor] = None,
                         rho_out: Optional[torch.Tensor] = None, workspace: Optional[torch.Tensor] = None):
    """feat: bf16 [N, D] preview embeddings on the GPU.  Returns (rho [3] = rho_g, rho_d, rho;
    d [N])."""
    if feat.dtype != torch.bfloat16 or feat.dim() != 2:
        raise PaceError("feat must be a 2-D bfloat16 tensor")
    N, D = feat.shape
    dev = feat.device
    if d_out is None:
        d_out = torch.empty(N, dtype=torch.float32, device=dev)
    if rho_out is None:
        rho_out = torch.empty(3, dtype=torch.float32, device=dev)
    if workspace is None:
        workspace = _ws(lib().pace_apc_density_features_workspace_size(N, D), dev)
    _check(lib().pace_apc_density_features(_ptr(feat), N, D, float(tail_frac), float(alpha),
                                           float(gamma), _ptr(d_out), _ptr(rho_out), _ptr(workspace),
                                           workspace.numel(), _stream()), "pace_apc_density_features")
    return rho_out, d_out


PIXEL_STATISTICS = {"rgb": 0, "entropy": 1, "edges": 2, "laplacian": 3}


def pixel_feature_dim(kind: int, patch: int) -> int:
    return (6, 64, 8, patch * patch)[kind]


def apc_pixel_features(img: torch.Tensor, kind: int, patch: int = 14,
                       out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """img: uint8 [H, W, 3] on the GPU.  Returns fp32 [N, dim] pixel-statistic preview vectors."""
    if img.dtype != torch.uint8 or img.dim() != 3 or img.shape[2] != 3:
        raise PaceError("img must be a uint8 [H, W, 3] tensor")
    H, W, _ = img.shape
    if not 0 <= kind <= 3:
        raise PaceError(f"kind={kind} not in 0..3")
    N = (H // patch) * (W // patch)
    if out is None:
        out = torch.empty(N, pixel_feature_dim(kind, patch), dtype=torch.float32, device=img.device)
    _check(lib().pace_apc_pixel_features(_ptr(img), H, W, patch, kind, _ptr(out), _stream()),
           "pace_apc_pixel_features")
    return out


def apc_pixel_density(img: torch.Tensor, kind: int, patch: int = 14, tail_frac: float = 0.10,
                      alpha: float = 0.6, gamma: float = 1.5, d_out: Optional[torch.Tensor] = None,
                      rho_out: Optional[torch.Tensor] = None, workspace: Optional[torch.Tensor] = None):
    """APC density with a pixel-statistic preview.  Returns (rho [3]: rho_g, rho_d, rho; d [N])."""
    if img.dtype != torch.uint8 or img.dim() != 3 or img.shape[2] != 3:
        raise PaceError("img must be a uint8 [H, W, 3] tensor")
    H, W, _ = img.shape
    N = (H // patch) * (W // patch)
    dev = img.device
    if d_out is None:
        d_out = torch.empty(max(N, 1), dtype=torch.float32, device=dev)
    if rho_out is None:
        rho_out = torch.empty(3, dtype=torch.float32, device=dev)
    if workspace is None:
        workspace = _ws(lib().pace_apc_pixel_density_workspace_size(H, W, patch, kind), dev)
    _check(lib().pace_apc_pixel_density(_ptr(img), H, W, patch, kind, float(tail_frac), float(alpha),
                                        float(gamma), _ptr(d_out), _ptr(rho_out), _ptr(workspace),
                                        workspace.numel(), _stream()), "pace_apc_pixel_density")
    return rho_out, d_out


class PreviewWeights(ctypes.Structure):
    """Mirror of pace_preview_weights (include/pace.h)."""
    _fields_ = [("pe", c_void), ("g1", c_void), ("wq", c_void), ("wk", c_void), ("wv", c_void),
                ("bq", c_void), ("bk", c_void), ("bv", c_void), ("wo", c_void), ("bo", c_void),
                ("g2", c_void), ("wgu", c_void), ("bgu", c_void), ("wd", c_void), ("bd", c_void),
                ("dim", c_int), ("ffn", c_int)]


def preview_weights_to_device(w: dict, device) -> dict:
    """Device copies of preview-block weights in the layout pace_apc_preview reads: bf16 bit
    arrays (uint16) and fp32 vectors as given; the patch embedding zero-padded to a multiple of
    8 columns, the hidden units zero-padded to a multiple of 8, gate and up rows interleaved.
    (Marshalling only: zero padding and row order leave the block's function unchanged.)"""
    import numpy as np

    def bf(a):
        return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).to(device)

    def f32(a):
        return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(device)

    D, kin = w["pe"].shape
    F = w["wg"].shape[0]
    kp = (kin + 7) // 8 * 8
    F8 = (F + 7) // 8 * 8
    pe = np.zeros((D, kp), np.uint16)
    pe[:, :kin] = w["pe"]
    wgu = np.zeros((2 * F8, D), np.uint16)
    wgu[0:2 * F:2] = w["wg"]
    wgu[1:2 * F:2] = w["wu"]
    bgu = np.zeros(2 * F8, np.float32)
    bgu[0:2 * F:2] = w["bg"]
    bgu[1:2 * F:2] = w["bu"]
    wd = np.zeros((D, F8), np.uint16)
    wd[:, :F] = w["wd"]
    out = {"pe": bf(pe), "wgu": bf(wgu), "bgu": f32(bgu), "wd": bf(wd), "dim": D, "ffn": F8}
    for k in ("wq", "wk", "wv", "wo"):
        out[k] = bf(w[k])
    for k in ("g1", "g2", "bq", "bk", "bv", "bo", "bd"):
        out[k] = f32(w[k])
    return out


def apc_preview(img: torch.Tensor, patch: int, token_patch: torch.Tensor, cu_windows: torch.Tensor,
                max_window: int, wdev: dict, out: Optional[torch.Tensor] = None,
                workspace: Optional[torch.Tensor] = None) -> torch.Tensor:
    """The preview block's token embeddings, bf16 [N, D]; wdev from preview_weights_to_device."""
    H, W, _ = img.shape
    N = (H // patch) * (W // patch)
    D, F = wdev["dim"], wdev["ffn"]
    dev = img.device
    if out is None:
        out = torch.empty((N, D), dtype=torch.bfloat16, device=dev)
    if workspace is None:
        workspace = _ws(lib().pace_apc_preview_workspace_size(N, D, F, patch), dev)
    pw = PreviewWeights(*(_ptr(wdev[k]) for k in ("pe", "g1", "wq", "wk", "wv", "bq", "bk", "bv", "wo", "bo",
                                                  "g2", "wgu", "bgu", "wd", "bd")), D, F)
    nwin = cu_windows.numel() - 1
    _check(lib().pace_apc_preview(_ptr(img), H, W, patch, _ptr(token_patch), _ptr(cu_windows), nwin,
                                  int(max_window), ctypes.byref(pw), _ptr(out), _ptr(workspace),
                                  workspace.numel(), _stream()), "pace_apc_preview")
    return out


def gemm_bf16(a: torch.Tensor, b: torch.Tensor, bias: Optional[torch.Tensor] = None,
              residual: Optional[torch.Tensor] = None, epilogue: int = 0,
              out: Optional[torch.Tensor] = None) -> torch.Tensor:
    """C = a b^T (+ bias, + residual, or SwiGLU of interleaved columns); a [M, K], b [N, K] bf16."""
    M, K = a.shape
    N = b.shape[0]
    if out is None:
        out = torch.empty((M, N // 2 if epilogue == 2 else N), dtype=torch.bfloat16, device=a.device)
    _check(lib().pace_gemm_bf16(_ptr(a), _ptr(b), _ptr(bias), _ptr(residual), _ptr(out), M, N, K, int(epilogue),
                                _stream()), "pace_gemm_bf16")
    return out


def apc_downsample(src: torch.Tensor, oH: int, oW: int, dst: Optional[torch.Tensor] = None):
    H, W, _ = src.shape
    if dst is None:
        dst = torch.empty((oH, oW, 3), dtype=torch.uint8, device=src.device)
    _check(lib().pace_apc_downsample(_ptr(src), H, W, _ptr(dst), oH, oW, _stream()),
           "pace_apc_downsample")
    return dst


# ---------------------------------------------------------------- attention
def vit_attention(q: torch.Tensor, k: torch.Tensor, v: torch.Tensor, cu_seqlens: torch.Tensor,
                  max_seglen: int, scale: Optional[float] = None, want_lse: bool = True,
                  want_mass: bool = True, o: Optional[torch.Tensor] = None,
                  lse: Optional[torch.Tensor] = None, mass: Optional[torch.Tensor] = None,
                  workspace: Optional[torch.Tensor] = None):
    """q, k, v: bf16 [N, H, d]; cu_seqlens int32 [nseg+1].  Returns (o, lse or None, mass or None)."""
    N, H, d = q.shape
    dev = q.device
    scale = 1.0 / math.sqrt(d) if scale is None else scale
    if o is None:
        o = torch.empty_like(q)
    if want_lse and lse is None:
        lse = torch.empty((H, N), dtype=torch.float32, device=dev)
    if want_mass and mass is None:
        mass = torch.empty((H, N), dtype=torch.float32, device=dev)
    if not want_lse:
        lse = None
    if not want_mass:
        mass = None
    nseg = cu_seqlens.numel() - 1
    if workspace is None:
        # the library needs a workspace for LSE scratch (mass without lse) and for the fp16 V^T
        # tiles of the long-segment kernel; the size says which applies
        need = lib().pace_vit_attention_workspace_size(N, H, d, nseg, int(max_seglen))
        lse_scratch = (N * H * 4 + 255) // 256 * 256
        if (mass is not None and lse is None) or need > lse_scratch:
            workspace = _ws(need, dev)
    _check(lib().pace_vit_attention(_ptr(q), _ptr(k), _ptr(v), N, H, d, _ptr(cu_seqlens),
                                    cu_seqlens.numel() - 1, int(max_seglen), float(scale), _ptr(o),
                                    _ptr(lse), _ptr(mass), _ptr(workspace),
                                    0 if workspace is None else workspace.numel(), _stream()),
           "pace_vit_attention")
    return o, lse, mass


def vit_attention_mass(q: torch.Tensor, k: torch.Tensor, cu_seqlens: torch.Tensor, max_seglen: int,
                       lse: torch.Tensor, scale: Optional[float] = None,
                       mass: Optional[torch.Tensor] = None):
    """Mass pass alone from a given LSE [H, N].  Returns mass fp32 [H, N]."""
    N, H, d = q.shape
    scale = 1.0 / math.sqrt(d) if scale is None else scale
    if mass is None:
        mass = torch.empty((H, N), dtype=torch.float32, device=q.device)
    _check(lib().pace_vit_attention_mass(_ptr(q), _ptr(k), N, H, d, _ptr(cu_seqlens),
                                         cu_seqlens.numel() - 1, int(max_seglen), float(scale),
                                         _ptr(lse), _ptr(mass), _stream()), "pace_vit_attention_mass")
    return mass


def prefill_attention_with_mass(q, k, v, cu_seqlens, max_seqlen: int, vis_len, cu_vis,
                                nvis_total: int, max_vis_len: int, mq_start, mq_len,
                                max_mq_len: int, scale: Optional[float] = None, want_mass=True,
                                o=None, lse=None, mass=None, workspace=None, vis_start=None):
    """Causal GQA prefill.  q bf16 [Ntot, Hq, d]; k, v bf16 [Ntot, Hkv, d]; metadata int32 on the
    GPU (vis_start None: visual tokens first).  Returns (o, lse [Hq, Ntot], mass [Hq, nvis_total]
    or None)."""
    Ntot, Hq, d = q.shape
    Hkv = k.shape[1]
    dev = q.device
    scale = 1.0 / math.sqrt(d) if scale is None else scale
    if o is None:
        o = torch.empty_like(q)
    if lse is None:
        lse = torch.empty((Hq, Ntot), dtype=torch.float32, device=dev)
    if want_mass and mass is None:
        mass = torch.empty((Hq, max(1, nvis_total)), dtype=torch.float32, device=dev)
    if not want_mass:
        mass = None
    _check(lib().pace_prefill_attention_with_mass(
        _ptr(q), _ptr(k), _ptr(v), Ntot, Hq, Hkv, d, _ptr(cu_seqlens), cu_seqlens.numel() - 1,
        int(max_seqlen), _ptr(vis_start), _ptr(vis_len), _ptr(cu_vis), int(nvis_total), int(max_vis_len),
        _ptr(mq_start), _ptr(mq_len), int(max_mq_len), float(scale), _ptr(o), _ptr(lse),
        _ptr(mass), _ptr(workspace), 0 if workspace is None else workspace.numel(), _stream()),
        "pace_prefill_attention_with_mass")
    return o, lse, mass


# ---------------------------------------------------------------- DDAE
def ddae_select(vis_mass: torch.Tensor, merge: int, vis_perm: Optional[torch.Tensor],
                llm_mass: torch.Tensor, nv: Sequence[int], keep: Sequence[int], mode: int = 0,
                tau: float = 0.5, w_llm_fixed: float = 0.5, hidden: Optional[torch.Tensor] = None,
                idx_out=None, score_out=None, fuse_out=None, out=None, workspace=None):
    """Segmented DDAE selection.  vis_mass fp32 [Hv, sum(nv)*merge]; llm_mass fp32 [Hl, sum(nv)];
    nv, keep: host lists.  Returns (idx int32 [sum keep], scores fp32 [sum nv], fuse fp32 [B, 4],
    gathered rows or None)."""
    B = len(nv)
    dev = llm_mass.device
    nv_total = int(sum(nv))
    ktot = int(sum(keep))
    Hv = vis_mass.shape[0]
    Hl = llm_mass.shape[0]
    if idx_out is None:
        idx_out = torch.empty(max(1, ktot), dtype=torch.int32, device=dev)
    if score_out is None:
        score_out = torch.empty(nv_total, dtype=torch.float32, device=dev)
    if fuse_out is None:
        fuse_out = torch.empty((B, 4), dtype=torch.float32, device=dev)
    row_bytes = 0
    if hidden is not None:
        row_bytes = hidden[0].numel() * hidden.element_size()
        if out is None:
            out = torch.empty((max(1, ktot),) + tuple(hidden.shape[1:]), dtype=hidden.dtype, device=dev)
    if workspace is None:
        workspace = _ws(lib().pace_ddae_select_workspace_size(nv_total, B), dev)
    nv_a = (ctypes.c_int * B)(*[int(x) for x in nv])
    kp_a = (ctypes.c_int * B)(*[int(x) for x in keep])
    _check(lib().pace_ddae_select_varlen(
        _ptr(vis_mass), Hv, merge, _ptr(vis_perm), _ptr(llm_mass), Hl, B, nv_a, kp_a, int(mode),
        float(tau), float(w_llm_fixed), _ptr(hidden), row_bytes, _ptr(idx_out), _ptr(score_out),
        _ptr(fuse_out), _ptr(out), _ptr(workspace), workspace.numel(), _stream()),
        "pace_ddae_select_varlen")
    return idx_out[:ktot], score_out, fuse_out, (out[:ktot] if out is not None else None)


def ddae_select_noalloc(vis_mass: torch.Tensor, merge: int, vis_perm: Optional[torch.Tensor],
                        llm_mass: torch.Tensor, nv: Sequence[int], keep: Sequence[int], mode: int = 0,
                        tau: float = 0.5, w_llm_fixed: float = 0.5, hidden: Optional[torch.Tensor] = None,
                        idx_out=None, score_out=None, fuse_out=None, out=None):
    """pace_ddae_select_varlen_noalloc: ddae_select without a workspace (the library's static
    per-GPU scratch); outputs are the caller's tensors, allocated here only when not given."""
    B = len(nv)
    dev = llm_mass.device
    nv_total = int(sum(nv))
    ktot = int(sum(keep))
    if idx_out is None:
        idx_out = torch.empty(max(1, ktot), dtype=torch.int32, device=dev)
    if score_out is None:
        score_out = torch.empty(nv_total, dtype=torch.float32, device=dev)
    if fuse_out is None:
        fuse_out = torch.empty((B, 4), dtype=torch.float32, device=dev)
    row_bytes = 0
    if hidden is not None:
        row_bytes = hidden[0].numel() * hidden.element_size()
        if out is None:
            out = torch.empty((max(1, ktot),) + tuple(hidden.shape[1:]), dtype=hidden.dtype, device=dev)
    nv_a = (ctypes.c_int * B)(*[int(x) for x in nv])
    kp_a = (ctypes.c_int * B)(*[int(x) for x in keep])
    _check(lib().pace_ddae_select_varlen_noalloc(
        _ptr(vis_mass), vis_mass.shape[0], merge, _ptr(vis_perm), _ptr(llm_mass), llm_mass.shape[0], B, nv_a,
        kp_a, int(mode), float(tau), float(w_llm_fixed), _ptr(hidden), row_bytes, _ptr(idx_out),
        _ptr(score_out), _ptr(fuse_out), _ptr(out), _stream()), "pace_ddae_select_varlen_noalloc")
    return idx_out[:ktot], score_out, fuse_out, (out[:ktot] if out is not None else None)


def ddae_select_one(vis_mass, merge, vis_perm, llm_mass, K: int, mode=0, tau=0.5, w_llm_fixed=0.5,
                    hidden=None, workspace=None):
    """Single-image pace_ddae_select."""
    Nv = llm_mass.shape[1]
    dev = llm_mass.device
    idx = torch.empty(max(1, K), dtype=torch.int32, device=dev)
    sc = torch.empty(Nv, dtype=torch.float32, device=dev)
    fz = torch.empty(4, dtype=torch.float32, device=dev)
    out = None
    row_bytes = 0
    if hidden is not None:
        row_bytes = hidden[0].numel() * hidden.element_size()
        out = torch.empty((max(1, K),) + tuple(hidden.shape[1:]), dtype=hidden.dtype, device=dev)
    if workspace is None:
        workspace = _ws(lib().pace_ddae_select_workspace_size(Nv, 1), dev)
    _check(lib().pace_ddae_select(_ptr(vis_mass), vis_mass.shape[0], merge, _ptr(vis_perm),
                                  _ptr(llm_mass), llm_mass.shape[0], Nv, int(mode), float(tau),
                                  float(w_llm_fixed), int(K), _ptr(hidden), row_bytes, _ptr(idx),
                                  _ptr(sc), _ptr(fz), _ptr(out), _ptr(workspace), workspace.numel(),
                                  _stream()), "pace_ddae_select")
    return idx[:K], sc, fz, (out[:K] if out is not None else None)


def topk_gather(scores: torch.Tensor, K: int, hidden: Optional[torch.Tensor] = None):
    N = scores.numel()
    dev = scores.device
    idx = torch.empty(max(1, K), dtype=torch.int32, device=dev)
    out = None
    row_bytes = 0
    if hidden is not None:
        row_bytes = hidden[0].numel() * hidden.element_size()
        out = torch.empty((max(1, K),) + tuple(hidden.shape[1:]), dtype=hidden.dtype, device=dev)
    _check(lib().pace_topk_gather(_ptr(scores), N, int(K), _ptr(hidden), row_bytes, _ptr(idx),
                                  _ptr(out), None, 0, _stream()), "pace_topk_gather")
    return idx[:K], (out[:K] if out is not None else None)


def gather_rows(src: torch.Tensor, idx: torch.Tensor, out: Optional[torch.Tensor] = None):
    """out[r] = src[idx[r]] (whole rows, bit for bit); src [rows, ...] with 16-byte rows."""
    n = idx.numel()
    if out is None:
        out = torch.empty((n,) + tuple(src.shape[1:]), dtype=src.dtype, device=src.device)
    row_bytes = src[0].numel() * src.element_size() if src.shape[0] > 0 else 0
    _check(lib().pace_gather_rows(_ptr(src), src.shape[0], row_bytes, _ptr(idx), n, _ptr(out),
                                  _stream()), "pace_gather_rows")
    return out
