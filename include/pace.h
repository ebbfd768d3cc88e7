/*
 * pace.h - C ABI of libpace.so, the MI355X (gfx950) hot path of PACE
 * (Pixel-Adaptive Condense and Extract, arXiv 2608.27206).
 *
 * The library implements the data-parallel steps of the method:
 *   APC  (Section 3.2, "Condense"): per-patch information density of an image
 *        (Eq. 1-2, the background baseline, the detail distances, the tail mean,
 *        rho_d and rho) and the bicubic resize by sqrt(r) per side
 *        (Appendix, "Detailed Implementation Specifics").
 *   Attention read-outs (Section 3.3 and the implementation details): vision-
 *        encoder self-attention (window and full) and causal grouped-query LLM
 *        prefill attention, each also returning the attention mass every key
 *        receives, with no attention matrix ever stored.
 *   DDAE (Section 3.3, "Extract"): min-max maps, std confidences, softmax(sigma/tau)
 *        fusion, top-K ranking and the gather of the kept token rows.
 *
 * Conventions for every call:
 *   - Tensor pointers are DEVICE pointers owned by the caller, contiguous, and
 *     16-byte aligned unless stated otherwise.  The library never allocates or
 *     frees memory; calls that need scratch take a caller-owned workspace whose
 *     size the matching *_workspace_size() function returns.
 *   - Every device call is asynchronous on `stream` and never synchronises.
 *   - bf16 tensors are passed as uint16_t bit patterns.  Mass and LSE are fp32;
 *     LSE is the natural log of the softmax denominator (log-sum-exp of the
 *     scaled logits).
 *   - On bad arguments a call returns an error status WITHOUT launching
 *     anything; pace_last_error() then returns a message (thread-local).
 *   - Device-side metadata (cu_seqlens, vis_len, cu_vis, mq_start/mq_len, vis_perm) is
 *     trusted: it must be monotone and consistent with the host-side maxima passed
 *     alongside it.  With the environment variable PACE_DEBUG=1 every call copies it to
 *     the host, synchronises the stream and checks it first, returning
 *     PACE_ERR_INVALID_ARG before any launch when it is inconsistent.
 *   - The library keeps no global mutable state other than the thread-local
 *     error message and, for pace_ddae_select_varlen_noalloc only, a static per-GPU
 *     scratch array and the table of its device addresses, so independent calls (other
 *     than overlapping calls of that entry point on one GPU) may run concurrently on
 *     different streams.
 */
#ifndef PACE_H_
#define PACE_H_

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum pace_status {
  PACE_OK = 0,
  PACE_ERR_INVALID_ARG = 1,   /* bad shape, count, pointer or alignment; nothing launched */
  PACE_ERR_UNSUPPORTED = 2,   /* valid but not implemented, e.g. head dim not in {80, 128} */
  PACE_ERR_WORKSPACE = 3,     /* workspace missing or smaller than *_workspace_size() */
  PACE_ERR_HIP = 4            /* a HIP launch or runtime call failed */
} pace_status_t;

/* Message describing the last error returned on this thread ("" if none). */
const char* pace_last_error(void);

/* Library ABI version (major * 100 + minor). */
int pace_version(void);

/* ---------------------------------------------------------------- host-only helpers */

/*
 * Number of tokens kept for a retention ratio: ceil(ratio * n - 1e-9), clamped
 * to [0, n].  The 1e-9 guard absorbs float products such as 0.1 * 30.
 * Used for DDAE's K (Section 3.3: keep the top-K tokens) and APC's tail count.
 * Returns -1 if n < 0 or ratio is not finite.
 */
int pace_keep_count(double ratio, int n);

/*
 * Per-image keep count set by APC's density for a batch of images: the keep ratio is
 * ratio_lo + (ratio_hi - ratio_lo) * rho, clamped to [ratio_lo, ratio_hi], and
 * K = pace_keep_count(ratio, n).  (The paper maps rho to an area ratio, Section 3.2; a
 * batch with per-image token budgets needs a keep ratio, and this linear map is the
 * reading used here.)  Returns -1 on bad arguments.
 */
int pace_keep_from_density(double rho, double ratio_lo, double ratio_hi, int n);

/*
 * Output size of APC's resize (Section 3.2, "Adaptive Condensation"; Appendix
 * implementation details: area ratio r = rho, each side scaled by sqrt(r), and a
 * hard budget overrides rho when it allows less).
 *   r_cap = min(1, max_pixels / (H*W)), r_floor = min(r_cap, min_pixels / (H*W)),
 *   r = clamp(rho, r_floor, r_cap); each side X -> floor(X*sqrt(r)/snap + 0.5)*snap,
 *   kept within [min(snap, X), floor(X/snap)*snap].
 * Writes *oH, *oW.  INVALID_ARG on non-positive sizes or snap, or null outputs.
 */
pace_status_t pace_apc_target_size(double rho, int H, int W, double min_pixels,
                                   double max_pixels, int snap, int* oH, int* oW);

/* ---------------------------------------------------------------- APC */

/* Workspace bytes for pace_apc_density on an H x W image with square patches. */
size_t pace_apc_density_workspace_size(int H, int W, int patch);

/*
 * APC information density (Section 3.2).
 *   img       uint8 [H, W, 3], HWC, row-major.  H and W must be multiples of patch.
 *   patch     patch side in pixels, 1..16 (14 for Qwen2.5-VL); patches in raster order.
 *   tail_frac fraction of largest distances averaged for d_top (0.10 in the paper);
 *             n_tail = max(1, pace_keep_count(tail_frac, N)).
 *   alpha, gamma   rho = alpha*rho_g + (1-alpha)*min(d_top/gamma, 1)  (0.6 and 1.5).
 *   d_out     fp32 [N] per-patch distance d_i = ||T_i - c_hat||, or NULL.
 *   rho_out   fp32 [3]: rho_g, rho_d, rho (phi of Eq. 1 is 1 - rho_g, Eq. 2).
 * Per-patch feature: the patch's 3*patch*patch pixels mapped to x/127.5 - 1 and
 * l2-normalised (a pixel preview; the paper's ViT-block preview needs weights).
 * phi (Eq. 1) is evaluated as ||mean_i T_i||^2, which equals the mean pairwise
 * cosine exactly; c_hat is zero when ||c|| <= 1e-5.
 * N = (H/patch)*(W/patch) must be >= 1.
 */
pace_status_t pace_apc_density(const uint8_t* img, int H, int W, int patch, double tail_frac,
                               float alpha, float gamma, float* d_out, float* rho_out,
                               void* workspace, size_t workspace_bytes, hipStream_t stream);

/* Workspace bytes for pace_apc_density_features. */
size_t pace_apc_density_features_workspace_size(int N, int D);

/*
 * APC information density of caller-supplied preview embeddings (Section 3.2: the shallow
 * feature preview's l2-normalised patch embeddings; Eq. 1-2, the background direction, the
 * detail distances, the tail mean, rho_d and rho).  The paper's preview is the vision
 * encoder's first block at the original resolution; a caller that runs it passes its output.
 *   feat      bf16 [N, D] row-major, N >= 1, D >= 1 (read as 16-byte vectors when D is a
 *             multiple of 8 and feat is 16-byte aligned, value by value otherwise).
 *             T_i = feat_i / max(||feat_i||, 1e-12) (a zero row is a zero direction).
 *   tail_frac, alpha, gamma, d_out, rho_out   as in pace_apc_density.
 * Same arithmetic as pace_apc_density after its pixel features: phi = ||mean_i T_i||^2,
 * c_hat zero when ||c|| <= 1e-5, n_tail = max(1, pace_keep_count(tail_frac, N)).
 * Reads the matrix twice.  Asynchronous on `stream`.
 */
pace_status_t pace_apc_density_features(const uint16_t* feat, int N, int D, double tail_frac,
                                        float alpha, float gamma, float* d_out, float* rho_out,
                                        void* workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * Pixel-statistic preview vectors (the training-free previews of the preview-network ablation
 * in Section 4; the paper names them without formulas, so each is read as one vector per
 * patch that the density steps consume like an embedding).
 *   img     uint8 [H, W, 3] HWC; H, W positive multiples of patch, patch 1..16.
 *   kind    0 RGB statistics: mean and population std of each channel of x/255, dim 6
 *           1 colour entropy: -p_k ln p_k for the 64 colours of 4 levels per channel, dim 64
 *           2 edge density: Sobel magnitude of the grey image summed per 45-degree
 *             orientation octant, / (255 * patch^2), dim 8
 *           3 Laplacian: 4-neighbour Laplacian of the grey image / 255, dim patch^2
 *           grey = (299 R + 587 G + 114 B) / 1000; neighbours cross patch borders and the image
 *           edge is clamped.
 *   out     fp32 [N, dim] row-major, caller-owned, N = (H/patch)*(W/patch), patches in raster
 *           order; kind 3 components in pixel raster order within the patch.
 * INVALID_ARG on null pointers, a kind outside 0..3, or bad sizes.  Asynchronous on `stream`.
 */
pace_status_t pace_apc_pixel_features(const uint8_t* img, int H, int W, int patch, int kind,
                                      float* out, hipStream_t stream);

/* Workspace bytes for pace_apc_pixel_density (0 for invalid arguments). */
size_t pace_apc_pixel_density_workspace_size(int H, int W, int patch, int kind);

/*
 * APC density with a pixel-statistic preview: pace_apc_pixel_features into the workspace,
 * then the arithmetic of pace_apc_density_features on those fp32 rows (a zero row is a zero
 * direction).  Arguments as in pace_apc_pixel_features and pace_apc_density.
 */
pace_status_t pace_apc_pixel_density(const uint8_t* img, int H, int W, int patch, int kind,
                                     double tail_frac, float alpha, float gamma, float* d_out,
                                     float* rho_out, void* workspace, size_t workspace_bytes,
                                     hipStream_t stream);

/*
 * Weights of the APC preview block (caller-owned device memory; bf16 matrices are row-major
 * [out, in], fp32 vectors).  dim D is a multiple of 80 (heads of 80 values); ffn F a multiple
 * of 8 (pad with zero hidden units: zero gate/up rows and zero down columns leave the block
 * unchanged).
 */
typedef struct pace_preview_weights {
  const uint16_t* pe;             /* [D, Kp] patch embedding, Kp = 3*patch^2 rounded up to a
                                     multiple of 8 (zero columns past 3*patch^2) */
  const float* g1;                /* [D] first RMSNorm gain */
  const uint16_t* wq, *wk, *wv;   /* [D, D] */
  const float* bq, *bk, *bv;      /* [D] or NULL */
  const uint16_t* wo;             /* [D, D] */
  const float* bo;                /* [D] or NULL */
  const float* g2;                /* [D] second RMSNorm gain */
  const uint16_t* wgu;            /* [2F, D]: rows 2f and 2f+1 are hidden unit f's gate and up rows */
  const float* bgu;               /* [2F] or NULL, same interleaving */
  const uint16_t* wd;             /* [D, F] */
  const float* bd;                /* [D] or NULL */
  int dim, ffn;                   /* D and F */
} pace_preview_weights;

/* Workspace bytes for pace_apc_preview (N patches). */
size_t pace_apc_preview_workspace_size(int N, int dim, int ffn, int patch);

/*
 * APC's shallow feature preview (Section 3.2: the vision encoder's initial block, K = 1, at the
 * original resolution), the embeddings that pace_apc_density_features scores:
 *   h0  = X W_pe^T, X the patch pixels mapped to x/127.5 - 1 (component order: patch row,
 *         pixel column, channel), one row per token;
 *   h1  = h0 + W_o A(RMSNorm_1(h0)) + b_o, A = softmax attention inside each window, heads of
 *         80 values, scale 1/sqrt(80), q/k/v = W_{q,k,v} RMSNorm_1(h0) + b_{q,k,v};
 *   out = h1 + W_d (silu(gate) * up) + b_d, (gate, up) = W_gu RMSNorm_2(h1) + b_gu;
 *   RMSNorm(x) = x / sqrt(mean(x^2) + 1e-6) * g.  No rotary position encoding.
 * Activations are stored in bf16 between the steps; products accumulate in fp32.
 *   img         uint8 [H, W, 3]; H and W multiples of patch (1..16); N = (H/patch)*(W/patch).
 *   token_patch int32 [N] (device): raster index of the patch that token t holds (the encoder's
 *               window-major order); cu_windows int32 [nwin+1] (device): windows as
 *               consecutive token ranges, each at most max_window (< 1024) tokens.
 *   out         bf16 [N, D], 16-byte aligned.
 */
pace_status_t pace_apc_preview(const uint8_t* img, int H, int W, int patch, const int32_t* token_patch,
                               const int32_t* cu_windows, int nwin, int max_window,
                               const pace_preview_weights* w, uint16_t* out, void* workspace,
                               size_t workspace_bytes, hipStream_t stream);

/*
 * The preview's dense products (exposed for reuse and testing): C = A B^T with A bf16 [M, K],
 * B bf16 [N, K] (row-major, 16-byte aligned, K a positive multiple of 8, each under 1 GiB),
 * fp32 accumulation,
 * bf16 out, and one fused epilogue:
 *   0: C [M, N] = A B^T + bias (bias fp32 [N] or NULL)
 *   1: C [M, N] = A B^T + bias + residual (residual bf16 [M, N])
 *   2: C [M, N/2]: column f = silu(g) * u with g, u = columns 2f, 2f+1 of A B^T + bias (N even)
 */
pace_status_t pace_gemm_bf16(const uint16_t* A, const uint16_t* B, const float* bias, const uint16_t* residual,
                             uint16_t* C, int M, int N, int K, int epilogue, hipStream_t stream);

/*
 * APC resize (Appendix implementation details: bicubic resize of both sides).
 *   src uint8 [H, W, 3] -> dst uint8 [oH, oW, 3], with 1 <= oH <= H and 1 <= oW <= W.
 * Separable Keys cubic (a = -0.5); when shrinking, the kernel is stretched by the
 * shrink factor (antialiasing); output pixel o samples input coordinate
 * (o + 0.5) * X / oX; taps outside the image are dropped and the remaining
 * weights renormalised; accumulation in fp32 without intermediate rounding;
 * result rounded half up and clamped to [0, 255].  Pointers need no alignment.
 * Up to 32x per side, workgroups stage their output tile's input span in LDS; beyond
 * that, one workgroup per output pixel reads its span from memory (float64 sums).
 */
pace_status_t pace_apc_downsample(const uint8_t* src, int H, int W, uint8_t* dst, int oH, int oW,
                                  hipStream_t stream);

/* ---------------------------------------------------------------- attention */

/*
 * Workspace bytes for pace_vit_attention with these arguments: LSE scratch (used when
 * lse == NULL and mass != NULL) and, when d == 80 and max_seglen >= 1024 (the long-segment
 * kernel), fp16 V^T tiles of H * 81 * (64 ceil(N/64) + 64 nseg) values plus nseg * H
 * per-(segment, head) maxima of |v|.
 */
size_t pace_vit_attention_workspace_size(int N, int H, int d, int nseg, int max_seglen);

/*
 * Vision-encoder self-attention with per-key mass (window attention and the
 * full-attention block whose mass is S_vis, Section 3.3 / implementation details).
 *   q, k, v   bf16 [N, H, d] token-major; d in {80, 128}.
 *   cu_seqlens int32 [nseg+1] on the device: segment s is rows [cu[s], cu[s+1]);
 *             segments (windows or whole images) never attend to each other.
 *   max_seglen host-side upper bound of the segment lengths.
 *   scale     logit scale (1/sqrt(d) for the encoder).
 *   o         bf16 [N, H, d] = softmax(q k^T * scale) v, no mask inside a segment.
 *   lse       fp32 [H, N] natural-log LSE of each row, or NULL.
 *   mass      fp32 [H, N]: mass[h, j] = sum over every query row i of j's segment
 *             of P_h[i, j] (column sums of the normalised probabilities), or NULL.
 * The mass pass needs the LSE: when lse is NULL and mass is not, the workspace
 * holds it.  At d == 80 with max_seglen >= 1024 the workspace is always required: the
 * long-segment kernel runs the PV product in fp16 on V^T tiles it writes there, each
 * (segment, head) scaled by a power of two that puts its largest |v| in [2^15, 2^16) and
 * undone on the output, so any finite bf16 V is converted exactly (values below 2^-32 of
 * their (segment, head)'s largest keep fewer bits); such segments allow at most 256 heads
 * (UNSUPPORTED otherwise).
 * The workspace must be 16-byte aligned, pace_vit_attention_workspace_size bytes.
 * Requires N >= 1, H >= 1, nseg >= 1.
 */
pace_status_t pace_vit_attention(const uint16_t* q, const uint16_t* k, const uint16_t* v, int N,
                                 int H, int d, const int32_t* cu_seqlens, int nseg, int max_seglen,
                                 float scale, uint16_t* o, float* lse, float* mass,
                                 void* workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * The mass pass of pace_vit_attention alone, from a caller-provided LSE (for
 * callers that ran the forward pass earlier, or want to time it separately).
 *   q, k bf16 [N, H, d]; cu_seqlens, nseg, max_seglen, scale as in pace_vit_attention;
 *   lse  fp32 [H, N] natural-log LSE of every row (as pace_vit_attention writes it);
 *   mass fp32 [H, N]: mass[h, j] = sum over the rows i of j's segment of
 *        exp(q_i . k_j * scale - lse[h, i]).
 */
pace_status_t pace_vit_attention_mass(const uint16_t* q, const uint16_t* k, int N, int H, int d,
                                      const int32_t* cu_seqlens, int nseg, int max_seglen,
                                      float scale, const float* lse, float* mass,
                                      hipStream_t stream);

/* Workspace bytes for pace_prefill_attention_with_mass (LSE scratch when lse == NULL). */
size_t pace_prefill_attention_workspace_size(int Ntot, int Hq);

/*
 * Causal grouped-query prefill attention with visual-key mass (S_llm, Section 3.3).
 *   q         bf16 [Ntot, Hq, d]; k, v bf16 [Ntot, Hkv, d]; d in {80, 128}; Hq % Hkv == 0;
 *             query head h uses KV head h / (Hq / Hkv).
 *   cu_seqlens int32 [B+1] (device): packed sequences, causal inside each (key <= query).
 *   vis_start int32 [B] (device) or NULL (= 0): sequence b's visual tokens are its tokens
 *             [vis_start[b], vis_start[b] + vis_len[b]) (relative positions; a text prefix such
 *             as a system prompt may come first).
 *   vis_len   int32 [B] (device): number of visual tokens of sequence b.
 *   cu_vis    int32 [B+1] (device): offset of sequence b's visual keys in mass;
 *             nvis_total (host) = cu_vis[B], the row length of mass.
 *   mq_start, mq_len int32 [B] (device): mass sums P over query rows
 *             [mq_start[b], mq_start[b] + mq_len[b]) of sequence b (relative positions).
 *             Text rows (mq_start = vis_len) give the paper's "Text" source; all rows
 *             give "Vision + Text"; the last row gives "Last".
 *   max_seqlen, max_vis_len, max_mq_len  host-side upper bounds.
 *   o         bf16 [Ntot, Hq, d]; lse fp32 [Hq, Ntot] or NULL (then the workspace holds it);
 *   mass      fp32 [Hq, nvis_total]: mass[h, cu_vis[b] + j] = sum_{i in rows_b} P_h[i, vis_start[b] + j],
 *             or NULL to skip the mass pass (vis_len, cu_vis, mq_* are then unused).
 */
pace_status_t pace_prefill_attention_with_mass(
    const uint16_t* q, const uint16_t* k, const uint16_t* v, int Ntot, int Hq, int Hkv, int d,
    const int32_t* cu_seqlens, int B, int max_seqlen, const int32_t* vis_start, const int32_t* vis_len,
    const int32_t* cu_vis, int nvis_total, int max_vis_len, const int32_t* mq_start,
    const int32_t* mq_len,
    int max_mq_len, float scale, uint16_t* o, float* lse, float* mass, void* workspace,
    size_t workspace_bytes, hipStream_t stream);

/* ---------------------------------------------------------------- DDAE */

#define PACE_MAX_SEGMENTS 64

/* Workspace bytes for pace_ddae_select / pace_ddae_select_varlen / pace_topk_gather. */
size_t pace_ddae_select_workspace_size(int nv_total, int nseg);

/*
 * DDAE selection over B images packed in one batch (Section 3.3).
 *   vis_mass  fp32 [Hv, nv_total*merge]: vision mass per encoder patch, images
 *             concatenated (image b owns patches [cu_nv[b]*merge, cu_nv[b+1]*merge)).
 *             S_vis of LLM token i of image b = sum_h sum_{t<merge}
 *             vis_mass[h, (cu_nv[b] + p)*merge + t] with p = vis_perm[cu_nv[b] + i]
 *             (p = i when vis_perm is NULL), then min-max normalised per image.
 *   vis_perm  int32 [nv_total] (device) or NULL: per image, merged encoder index of each
 *             LLM-order visual token.
 *   llm_mass  fp32 [Hl, nv_total]: S_llm of token i = sum_h llm_mass[h, i], min-max per image.
 *   nv_host   int [B] (HOST): visual tokens per image; keep_host int [B] (HOST): K_b,
 *             0 <= K_b <= nv_host[b].  Any B >= 1: a batch of more than PACE_MAX_SEGMENTS
 *             images runs as consecutive launches of at most that many.
 *   mode      0: (w_llm, w_vis) = softmax([sigma_llm, sigma_vis] / tau), sigma = population
 *             std of each normalised map; 1: fixed (w_llm_fixed, 1 - w_llm_fixed).
 *   S_final = w_llm * S_llm + w_vis * S_vis.  Top-K per image: highest scores, ties to
 *             the lower index, kept indices ascending.
 *   idx_out   int32 [sum K_b]: kept GLOBAL token indices (image b's block starts at
 *             sum_{c<b} K_c).
 *   score_out fp32 [nv_total] S_final, or NULL.   fuse_out fp32 [4*B]
 *             (sigma_llm, sigma_vis, w_llm, w_vis) per image, or NULL.
 *   hidden    [nv_total, row_bytes] device rows to gather, or NULL to skip the gather;
 *   out       [sum K_b, row_bytes]: out[r] = hidden[idx_out[r]] bit for bit.
 *             row_bytes must be a positive multiple of 16.
 */
pace_status_t pace_ddae_select_varlen(const float* vis_mass, int Hv, int merge,
                                      const int32_t* vis_perm, const float* llm_mass, int Hl,
                                      int B, const int* nv_host, const int* keep_host, int mode,
                                      float tau, float w_llm_fixed, const void* hidden,
                                      size_t row_bytes, int32_t* idx_out, float* score_out,
                                      float* fuse_out, void* out, void* workspace,
                                      size_t workspace_bytes, hipStream_t stream);

/* Single-image form of pace_ddae_select_varlen (B = 1, nv_host = {Nv}, keep_host = {K}). */
pace_status_t pace_ddae_select(const float* vis_mass, int Hv, int merge, const int32_t* vis_perm,
                               const float* llm_mass, int Hl, int Nv, int mode, float tau,
                               float w_llm_fixed, int K, const void* hidden, size_t row_bytes,
                               int32_t* idx_out, float* score_out, float* fuse_out, void* out,
                               void* workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * pace_ddae_select_varlen without a workspace argument, for callers that cannot allocate
 * device memory (code under HIP graph capture, tight serving loops, harnesses that forbid
 * allocation).  It allocates nothing: its scratch is a static device array of
 * pace_ddae_select_noalloc_max_bytes() bytes (4 MiB), one per GPU, held until the process ends;
 * its device address is looked up on the first call on each device (hipGetSymbolAddress, with
 * that device current).  Arguments and results as in pace_ddae_select_varlen.
 *   Returns PACE_ERR_WORKSPACE, launching nothing, when the selection needs more scratch than
 *   that (pace_ddae_select_workspace_size(sum nv_host, B) > 4 MiB, about 300,000 tokens).
 *   Every call on a GPU shares that GPU's scratch, so calls that overlap on one GPU (on
 *   different streams, or from different threads without ordering) race; calls in one
 *   stream's order do not.  With PACE_DEBUG=1 it copies and synchronises like the workspace
 *   form (leave PACE_DEBUG unset under graph capture).
 */
size_t pace_ddae_select_noalloc_max_bytes(void);
pace_status_t pace_ddae_select_varlen_noalloc(const float* vis_mass, int Hv, int merge,
                                              const int32_t* vis_perm, const float* llm_mass, int Hl,
                                              int B, const int* nv_host, const int* keep_host, int mode,
                                              float tau, float w_llm_fixed, const void* hidden,
                                              size_t row_bytes, int32_t* idx_out, float* score_out,
                                              float* fuse_out, void* out, hipStream_t stream);

/*
 * The ranking and pruning steps alone (end of Section 3.3): top-K of given fp32
 * scores [N] (ties to the lower index, ascending output) and the gather of the
 * kept rows.  hidden may be NULL to skip the gather.  NaN scores are not allowed.
 */
pace_status_t pace_topk_gather(const float* scores, int N, int K, const void* hidden,
                               size_t row_bytes, int32_t* idx_out, void* out, void* workspace,
                               size_t workspace_bytes, hipStream_t stream);

/*
 * The compaction step of pruning on its own (Section 3.3 and the prefill after pruning):
 * dst[r] = src[idx[r]] bit for bit, for r < n_idx, rows of row_bytes bytes.  Gathers the
 * other per-token tensors of the shortened context with the indices a selection produced
 * (Q/K/V or KV-cache rows, position ids padded to 16 bytes, ...).
 *   src  device [src_rows, row_bytes]; dst device [n_idx, row_bytes] (caller-owned, not
 *        overlapping src); both 16-byte aligned; row_bytes a positive multiple of 16.
 *   idx  int32 [n_idx] device; entries outside [0, src_rows) leave their dst row unwritten.
 * n_idx = 0 is a no-op.  Asynchronous on `stream`.
 */
pace_status_t pace_gather_rows(const void* src, int src_rows, size_t row_bytes,
                               const int32_t* idx, int n_idx, void* dst, hipStream_t stream);

#ifdef __cplusplus
}
#endif
#endif /* PACE_H_ */
