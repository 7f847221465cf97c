/*
 * spider.h - C ABI of the MI355X (gfx950) implementation of SPIDER's
 * pruned-and-skipped multimodal prefill (multi-layer semantic token pruning,
 * Sec. 4.1, and adaptive sub-layer skipping, Sec. 4.2-4.3 / Algorithm 1).
 *
 * Conventions for every entry point:
 *   - All device buffers are owned by the caller.  The library never
 *     allocates or frees device memory; scratch space comes from a
 *     caller-provided workspace whose size is given by the matching
 *     *_workspace_size() query.  Host arrays are read before the call
 *     returns and may be freed afterwards.
 *   - Arguments are validated before any HIP call.  On error nothing is
 *     enqueued, outputs are untouched, a non-zero spider_status is returned
 *     and a thread-local message is available from spider_last_error().
 *     A failed kernel launch returns SPIDER_ERR_HIP.  Faults inside kernels
 *     surface at the caller's next synchronisation of the stream.
 *   - All device work is enqueued on `stream` (a hipStream_t; NULL means the
 *     default stream).  Calls are asynchronous unless stated otherwise.
 *   - Strides are in elements, not bytes.  Row-major everywhere.
 *   - Identical inputs give bitwise-identical outputs on the same GPU (no
 *     floating-point atomics).
 *   - Calls on distinct workspaces are independent; the library keeps no
 *     per-call state except the thread-local error message, the optional
 *     profiler and the per-thread pinned staging buffers used by the
 *     prefill calls to upload row tables and read back admission flags
 *     and codes.
 */
#ifndef SPIDER_H
#define SPIDER_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  SPIDER_OK = 0,
  SPIDER_ERR_INVALID_ARG = 1,  /* null pointer, negative size, bad enum     */
  SPIDER_ERR_SHAPE = 2,        /* inconsistent sizes (keep > n, cap small)  */
  SPIDER_ERR_UNSUPPORTED = 3,  /* valid but not implemented (e.g. dh != 128 in bf16) */
  SPIDER_ERR_WORKSPACE = 4,    /* workspace null or smaller than required   */
  SPIDER_ERR_HIP = 5           /* a HIP runtime call or launch failed       */
} spider_status;

typedef enum { SPIDER_F32 = 0, SPIDER_BF16 = 1 } spider_dtype;

/* Opaque stream handle: pass a hipStream_t (or NULL for the default stream). */
typedef void* spider_stream;

/* Message of the last failing call on this thread ("" if none). */
const char* spider_last_error(void);

/* ABI version (major * 100 + minor). */
int spider_version(void);

/* ------------------------------------------------------------------------
 * Token budget (Sec. 4.1.1-4.1.2).  Host only, no HIP call.
 * The anchor budget n*R*r of Sec. 4.1.1 is taken per tile as
 * n_anchor = floor(keep * r_num / r_den) in exact integer arithmetic and the
 * complementary budget n*R*(1-r) of Sec. 4.1.2 as n_cmp = keep - n_anchor.
 * Requires keep >= 0, r_den > 0, 0 <= r_num <= r_den.
 * ------------------------------------------------------------------------ */
spider_status spider_budget(int keep, int r_num, int r_den, int* n_anchor, int* n_cmp);

/* Budgets from a retention ratio R_v = rv_num / rv_den of an input-dependent
 * token count n (the setting used for Qwen3-VL in the appendix): keep =
 * floor(n * rv_num / rv_den) in exact integer arithmetic, then n_anchor and
 * n_cmp as spider_budget(keep, r_num, r_den).  Requires n >= 0, rv_den > 0,
 * 0 <= rv_num <= rv_den and spider_budget's conditions.  Host only. */
spider_status spider_budget_ratio(int n, int rv_num, int rv_den, int r_num, int r_den, int* keep,
                                  int* n_anchor, int* n_cmp);

/* ------------------------------------------------------------------------
 * spider_anchor_colmean - anchor scores of an encoder without [CLS]
 * (Sec. 4.1.1: the mean attention each patch token receives):
 *   a_out[g*n + j] = (1 / (H*n)) * sum_h sum_i attn[g, h, i, j]
 * with element (g,h,i,j) at attn[g*stride_g + h*stride_h + i*stride_row + j]
 * (query patch i, key patch j; device fp32, 16-byte aligned; n, the strides
 * multiples of 4).  fp32 accumulation in a fixed order (per head, 128-row
 * chunks summed by rows in ascending order within each of four interleaved
 * row sets; the chunk sums, numbered head-major, added in ascending order
 * within four interleaved sets, the sets combined pairwise), one IEEE
 * division: identical inputs give identical bits.  The result feeds spider_score with
 * cls_attn = NULL.  Limits: 1 <= n <= 4096, 1 <= H <= 1024, 1 <= G <= 65535.
 * Workspace: spider_anchor_colmean_workspace_size(G, H, n) bytes, 256-byte
 * aligned (chunk sums; contents on entry ignored).
 * ------------------------------------------------------------------------ */
size_t spider_anchor_colmean_workspace_size(int G, int H, int n);

/* ------------------------------------------------------------------------
 * spider_cls_attention - the [CLS] row of a ViT layer's self-attention rebuilt
 * from its CLS query and keys, for encoders that never store attention maps
 * (the row Sec. 4.1.1 averages over heads):
 *   attn_out[(g*H + h)*n_tok + j] = softmax over j of scale * q[g,h,:] . k[g,j,h,:]
 * with q element (g,h,c) at q[g*q_stride_g + h*dh + c] and k element (g,j,h,c)
 * at k[g*k_stride_g + j*k_stride_row + h*dh + c] (token 0 = [CLS]); dtype of q
 * and k bf16 or fp32 (device), output fp32 [G, H, n_tok] contiguous: pass it
 * to spider_score with attn_stride_h = n_tok, attn_stride_g = H*n_tok,
 * attn_col0 = 1.  fp32 arithmetic in a fixed order (dot products over c
 * ascending, the row maximum subtracted, exponentials summed per thread in
 * token order then in a fixed tree, one IEEE division per token).
 * Limits: dh <= 256, n_tok <= 4097, G, H <= 65535; dh and the strides
 * multiples of 4, q and k aligned to 4 elements.  No workspace.
 * ------------------------------------------------------------------------ */
spider_status spider_cls_attention(int G, int H, int dh, int n_tok, const void* q, int64_t q_stride_g,
                                   const void* k, int64_t k_stride_g, int64_t k_stride_row,
                                   spider_dtype dtype, float scale, float* attn_out, spider_stream stream);

spider_status spider_anchor_colmean(int G, int H, int n, const float* attn, int64_t stride_g,
                                    int64_t stride_h, int64_t stride_row, float* a_out,
                                    void* workspace, size_t workspace_bytes, spider_stream stream);

/* ------------------------------------------------------------------------
 * spider_score - MSV-Prune scoring of G independent tiles (Sec. 4.1, Eq. 1
 * and Eq. 3, Algorithm 1 stage 1).  For every tile g and patch i < n:
 *   a[g,i]       = (sum over heads h = 0..H-1, in order, in fp32, of
 *                   cls_attn[g,h,attn_col0+i]) / H                (Sec. 4.1.1)
 *   anchors      = the n_anchor patches with the largest a, ties to the
 *                  lower index (Eq. 1 read as Algorithm 1's top-nRr)
 *   cluster[g,i] = -1 for anchors; otherwise the K-means cluster of the
 *                  patch's last-layer feature (Sec. 4.1.2): Euclidean Lloyd
 *                  iterations on the raw rows of F^L (the last entry of
 *                  feats), centroids initialised at the non-anchor rows
 *                  floor(k*m/K) (m = non-anchor count, rows in ascending
 *                  patch order), at most kmeans_max_iter assignment passes
 *                  with early exit when no assignment changes, ties to the
 *                  lower cluster, empty clusters keep their centroid; fp32.
 *   m[g,i]       = max over anchors p of cos(F^L_i, F^L_p)   (0 if none)
 *   s[g,i]       = mean over j in the cluster of i of the Eq. 3 score
 *                  S_ij = sum over tapped layers l of cos(F^l_i, F^l_j)
 *                         + m_i + m_j,
 *                  +inf for anchors.  Cosine with a zero row is 0.
 * Inputs:
 *   cls_attn  device fp32; element (g,h,c) at cls_attn[g*attn_stride_g +
 *             h*attn_stride_h + c]; patch i is column attn_col0 + i (the CLS
 *             row of the last tapped layer's attention, column 0 = CLS).
 *             NULL (with H = 0, strides and attn_col0 ignored): a_out holds
 *             the anchor scores on entry (e.g. from spider_anchor_colmean for
 *             encoders without [CLS]) and is left unchanged.
 *   feats     HOST array of n_layers device pointers (tapped layers, the last
 *             one is F^L), each of dtype feat_dtype; patch i of tile g is row
 *             feat_row0 + i: element (g,row,c) at feats[l][g*feat_stride_g +
 *             row*feat_stride_row + c].
 *   Limits: 1 <= n <= 4096, 1 <= H (0 with given scores), 1 <= d_v <= 2048, 1 <= n_layers <= 8,
 *   1 <= K <= 8, 0 <= n_anchor <= n, kmeans_max_iter >= 1.
 * Outputs (device, [G,n], row stride n): a_out fp32, cluster_out int32,
 *   s_out fp32, m_out fp32 (may be NULL).
 * Workspace: spider_score_workspace_size(G, n, d_v, n_layers, K) bytes,
 *   256-byte aligned device memory; contents on entry are ignored.
 * ------------------------------------------------------------------------ */
size_t spider_score_workspace_size(int G, int n, int d_v, int n_layers, int K);

spider_status spider_score(int G, int n, int H, int d_v, int n_layers,
                           const float* cls_attn, int64_t attn_stride_g,
                           int64_t attn_stride_h, int attn_col0,
                           const void* const* feats, spider_dtype feat_dtype,
                           int64_t feat_stride_g, int64_t feat_stride_row, int feat_row0,
                           int n_anchor, int K, int kmeans_max_iter,
                           float* a_out, int32_t* cluster_out, float* s_out, float* m_out,
                           void* workspace, size_t workspace_bytes, spider_stream stream);

/* ------------------------------------------------------------------------
 * spider_score_noalloc - spider_score without a workspace argument, for
 * callers that cannot allocate device memory (code under HIP graph capture,
 * tight serving loops, harnesses that forbid hipMalloc).  Arguments, outputs,
 * limits and results are those of spider_score (bit-identical outputs); the
 * scratch space is a static device array of SPIDER_SCORE_SCRATCH_BYTES that
 * every GPU the library runs on holds until the process ends.  Sizes whose
 * spider_score_workspace_size exceeds it are rejected with
 * SPIDER_ERR_WORKSPACE before any HIP call (e.g. 32 MiB holds about 50 tiles
 * of 576 patches with two tapped layers of width 1024 and K = 4).  The call
 * allocates nothing (no hipMalloc / hipFree); its first call on a device looks
 * up that device's scratch address.  All calls on one GPU share its scratch:
 * calls that overlap on one GPU (concurrent streams, or other host threads)
 * race and must be serialised by the caller; a later call on the same stream
 * is ordered after an earlier one and needs nothing.
 * ------------------------------------------------------------------------ */
#define SPIDER_SCORE_SCRATCH_BYTES (32u << 20)

spider_status spider_score_noalloc(int G, int n, int H, int d_v, int n_layers,
                                   const float* cls_attn, int64_t attn_stride_g,
                                   int64_t attn_stride_h, int attn_col0,
                                   const void* const* feats, spider_dtype feat_dtype,
                                   int64_t feat_stride_g, int64_t feat_stride_row, int feat_row0,
                                   int n_anchor, int K, int kmeans_max_iter,
                                   float* a_out, int32_t* cluster_out, float* s_out, float* m_out,
                                   spider_stream stream);

/* ------------------------------------------------------------------------
 * spider_select - quotas, complementary selection, spatial-order union
 * (Sec. 4.1.2, Eq. 2; Sec. 4.1) and optional assembly of the decoder input.
 * Per tile g (cluster/s as written by spider_score, row stride n):
 *   |C_k|   = number of patches with cluster == k (k < K);
 *   N_k     = quota_mode 0 (Eq. 2 literally): 0 for an empty cluster, else
 *             min(|C_k|, max(1, round_half_even(n_cmp*|C_k| / sum_j |C_j|)))
 *             computed exactly in integers (the total may differ from n_cmp);
 *             quota_mode 1: largest-remainder apportionment of exactly
 *             min(n_cmp, sum|C_j|) tokens, ties to the lower cluster;
 *             all quotas are 0 when n_cmp == 0;
 *   kept    = anchors (cluster == -1) plus, per cluster, the N_k patches
 *             with the smallest s (ties to the lower index; -0.0 == +0.0);
 *   idx_out[g, 0..count-1] = kept patch indices ascending; the rest of the
 *             row (up to cap) is -1; count_out[g] = count.
 *   cap must be >= min(n, n_anchor + n_cmp + K) (the largest count Eq. 2 can
 *   produce when n_anchor patches are anchors).
 * Assembly (skipped when src and x_out are both NULL): B = G / tiles_per_sample
 *   samples; the packed decoder input x_out holds, per sample b, the kept rows
 *   of its tiles in tile order (row i of tile g = src[g*src_stride_g +
 *   i*d_model]) followed by its n_text text rows (text[b*n_text*d_model +
 *   t*d_model]), samples one after another; cu_seqlens_out[0..B] (device
 *   int32) gets the sample boundaries.  With src == NULL and x_out given only
 *   the text rows and the boundaries are written: the kept rows are then
 *   projected into place by spider_project_kept.  src/text/x_out have dtype
 *   act_dtype.  x_out must hold B*(tiles_per_sample*cap + n_text) rows of
 *   d_model.  In quota_mode 0 the
 *   caller reads cu_seqlens_out (one device-to-host copy) to size the
 *   prefill; in quota_mode 1 every count is n_anchor + min(n_cmp, n - n_anchor).
 * No workspace.  Limits: 1 <= n <= 4096, 1 <= K <= 8, tiles_per_sample >= 1
 * dividing G, d_model % 8 == 0 when assembling.
 * ------------------------------------------------------------------------ */
spider_status spider_select(int G, int n, const int32_t* cluster, const float* s,
                            int n_anchor, int n_cmp, int K, int quota_mode,
                            int32_t* idx_out, int32_t* count_out, int cap,
                            int tiles_per_sample, const void* src, int64_t src_stride_g,
                            int d_model, spider_dtype act_dtype, const void* text, int n_text,
                            void* x_out, int32_t* cu_seqlens_out, spider_stream stream);

/* ------------------------------------------------------------------------
 * spider_project_kept - the multimodal projector on the kept rows only
 * (pruning happens in the ViT feature space, before the projector: the
 * appendix's reading for LLaVA and its AnyRes tiles).  For every tile g and
 * slot r < count[g] (idx, count as written by spider_select, idx row stride
 * cap), with x the feature row of patch idx[g*cap + r] (element (g,row,c) at
 * feats[g*feat_stride_g + row*feat_stride_row + c], patch i in row
 * feat_row0 + i):
 *   x_out[dst] = W2 GELU(W1 x + b1) + b2,   GELU(t) = t (1 + erf(t/sqrt 2)) / 2
 * where dst is the row spider_select's assembly gives that kept token (kept
 * rows of a sample's tiles in tile order, then its n_text text rows).
 * W1 [d_hid, d_in], W2 [d_out, d_hid] in nn.Linear layout and dtype; b1 [d_hid],
 * b2 [d_out] fp32 or NULL (zero).  Precision (bf16): GEMMs accumulate in fp32,
 * bias and GELU in fp32, the hidden rows and the outputs rounded to bf16;
 * (fp32): everything fp32.  Slots past count[g] are computed on a valid row
 * and never stored.  Requires feat_stride_g to be a multiple of
 * feat_stride_row; bf16: d_in, d_hid, d_out multiples of 64, feats/W1/W2
 * 16-byte aligned, feat_stride_row a multiple of 8.
 * Workspace: spider_project_kept_workspace_size(G, cap, d_hid, d_out, dtype).
 * ------------------------------------------------------------------------ */
size_t spider_project_kept_workspace_size(int G, int cap, int d_hid, int d_out, spider_dtype dtype);

spider_status spider_project_kept(int G, int tiles_per_sample, int cap, const int32_t* idx,
                                  const int32_t* count, const void* feats, int64_t feat_stride_g,
                                  int64_t feat_stride_row, int feat_row0, int d_in, const void* w1,
                                  const float* b1, int d_hid, const void* w2, const float* b2, int d_out,
                                  int n_text, spider_dtype dtype, void* x_out, void* workspace,
                                  size_t workspace_bytes, spider_stream stream);

/* ------------------------------------------------------------------------
 * Offline sub-layer contribution policy (Sec. 4.2.2, Eq. 5).  Host only.
 *   norm_f(l) = 1 - (slc_f(l) - min_l slc_f) / (max_l slc_f - min_l slc_f + eps)
 * for each family f in {attention, FFN}, in double precision; the per-layer
 * skip target is target_out[l] = 1 (FFN) if norm_ffn(l) > norm_attn(l) else
 * 0 (attention: ties go to attention), and slc_sel_out[l] = norm of that
 * target.  slc_attn/slc_ffn: host [L] floats.  Outputs host [L].
 * ------------------------------------------------------------------------ */
spider_status spider_slc_policy(int L, const float* slc_attn, const float* slc_ffn, double eps,
                                double* slc_sel_out, uint8_t* target_out);

/* ------------------------------------------------------------------------
 * spider_plan_skips - admission rule of Algorithm 1 / Eq. 6 for one sample.
 * Host only.  For layers l = 0 .. floor(L/2)-1 (the decision window,
 * 1-indexed l <= L/2) and every visual token i not yet in skip mode:
 *   acc_i += w1 * s_sa[l*s_sa_stride + i] + w2 * slc_sel[l]   (double)
 *   if acc_i >= T_skip: token i enters skip mode at layer l with its target
 *   frozen to target[l] (0 attention, 1 FFN).
 * A token admitted at layer l bypasses its target in layers l .. L-1:
 *   codes_out[l2*codes_stride + i] = 1 (attention) or 2 (FFN), else 0.
 * admit_out (may be NULL) receives the admission layer or -1.
 * s_sa: host [floor(L/2), s_sa_stride] floats; slc_sel: host [L] doubles;
 * target: host [L] bytes; codes_out: host [L, codes_stride] bytes.
 * ------------------------------------------------------------------------ */
spider_status spider_plan_skips(int L, int n_vis, const float* s_sa, int s_sa_stride,
                                const double* slc_sel, const uint8_t* target,
                                double w1, double w2, double T_skip,
                                uint8_t* codes_out, int codes_stride, int32_t* admit_out);

/* ------------------------------------------------------------------------
 * spider_prefill - LLaMA-style decoder prefill over packed samples with
 * per-row sub-layer bypass (VSkip-Attn / VSkip-FFN of Sec. 3.2, the forward
 * step of Algorithm 1).  Per layer l and row r (codes[l*rows + r]):
 *   bit 0 clear: h_r += Wo * Attn(RMSNorm(h; attn_norm))_r   (row is a query)
 *   bit 1 clear: h_r += Wd (silu(Wg x) * (Wu x)), x = RMSNorm(h; ffn_norm)_r
 * A row with bit 0 set gets no attention update but still provides keys and
 * values (computed from its current h); a row with bit 1 set gets no FFN
 * update; a bypassed row keeps its value exactly.  Attention is causal within
 * each sample (rows cu_seqlens[b] .. cu_seqlens[b+1]-1, positions restarting
 * at 0), multi-head with dh = d/H, scale 1/sqrt(dh), rotate-half RoPE with
 * base theta on queries and keys.  RMSNorm(x) = x / sqrt(mean(x^2) + eps) * w.
 * No work is launched for bypassed rows; a sub-layer with no active row in
 * a layer launches nothing (keys/values are not computed when no row of any
 * sample is a query).
 * Precision (dtype SPIDER_BF16): weights, x and activations bf16; residual h
 *   fp32; RMSNorm outputs, Q/K after RoPE, V, attention outputs and
 *   silu(g)*u rounded to bf16 (round-to-nearest-even) from fp32; GEMMs
 *   accumulate in fp32 (MFMA); O and down outputs are added to h in fp32;
 *   softmax in fp32.  Requires dh == 128, d % 64 == 0, d_ff % 64 == 0.
 * dtype SPIDER_F32: everything fp32 (any dh <= 256 with dh even).
 * Both: d % 4 == 0, d <= 8192; x (bf16), weights, norms and h_out 16-byte
 * aligned.
 * Inputs: cfg; layers = HOST array [L] of per-layer device weight pointers
 *   (matrices in nn.Linear layout [out, in], norms fp32 [d]); cu_seqlens =
 *   HOST int32 [B+1] (cu[0] = 0, non-decreasing); x = device [rows, d] in
 *   cfg->dtype with rows = cu_seqlens[B]; codes = HOST uint8 [L, rows].
 * Output: h_out device fp32 [rows, d] (the residual stream after layer L-1,
 *   before any final norm).  x and h_out must not overlap.
 * Workspace: spider_prefill_workspace_size(cfg, B, rows) bytes.
 * ------------------------------------------------------------------------ */
typedef struct {
  int L;            /* decoder layers                      */
  int d;            /* model width                         */
  int H;            /* attention heads (dh = d / H)        */
  int d_ff;         /* SwiGLU hidden width                 */
  float eps;        /* RMSNorm epsilon                     */
  float theta;      /* RoPE base                           */
  spider_dtype dtype;
} spider_decoder_cfg;

typedef struct {
  const float* attn_norm;   /* [d] fp32                    */
  const void* wq;           /* [d, d]                      */
  const void* wk;           /* [d, d]                      */
  const void* wv;           /* [d, d]                      */
  const void* wo;           /* [d, d]                      */
  const float* ffn_norm;    /* [d] fp32                    */
  const void* wg;           /* [d_ff, d]                   */
  const void* wu;           /* [d_ff, d]                   */
  const void* wd;           /* [d, d_ff]                   */
} spider_layer_weights;

size_t spider_prefill_workspace_size(const spider_decoder_cfg* cfg, int B, int rows);

/* KV cache of the decoder: keys after RoPE and values of every layer, in
 * cfg->dtype, layout [L][B][cap][d]: token at position p of sample b in layer l
 * at ((l*B + b)*cap + p)*d.  Device memory owned by the caller. */
typedef struct {
  void* k;
  void* v;
  int cap;          /* token slots per sample */
} spider_kv_cache;

spider_status spider_prefill(const spider_decoder_cfg* cfg, const spider_layer_weights* layers,
                             int B, const int32_t* cu_seqlens, const void* x,
                             const uint8_t* codes, float* h_out,
                             void* workspace, size_t workspace_bytes, spider_stream stream);

/* ------------------------------------------------------------------------
 * spider_prefill_kv - spider_prefill that also fills the KV cache a decode
 * step reads (the cache the pruned and skipped prefill leaves; Sec. 5 reports
 * decode over it): for every layer and every row (also rows that bypass
 * attention, whose keys and values later tokens still read) its key after
 * RoPE and its value, exactly the values the prefill's attention used, at
 * position 0.. of its sample.  Keys and values are produced in every layer,
 * also where no prefill row is a query.  Arguments and workspace as
 * spider_prefill, plus kv (every sample must fit: cu_seqlens[b+1] -
 * cu_seqlens[b] <= kv->cap; bf16 cache 16-byte aligned).
 * ------------------------------------------------------------------------ */
spider_status spider_prefill_kv(const spider_decoder_cfg* cfg, const spider_layer_weights* layers, int B,
                                const int32_t* cu_seqlens, const void* x, const uint8_t* codes,
                                float* h_out, const spider_kv_cache* kv, void* workspace,
                                size_t workspace_bytes, spider_stream stream);

/* ------------------------------------------------------------------------
 * spider_decode_step - one autoregressive step over the KV cache, then the LM
 * head (Algorithm 1 ends with it).  Sample b's new token (input row x[b],
 * device [B, d] in cfg->dtype) sits at position lens[b] (HOST int32 [B]:
 * tokens already in sample b's cache, 0 <= lens[b] < kv->cap, lens[b] < 8192);
 * it runs through every layer with nothing bypassed (same block, precision
 * and RoPE as spider_prefill), its key and value are written into the cache
 * at lens[b], and its query attends to cache positions 0..lens[b] (softmax and
 * P.V in fp32).  The caller advances lens afterwards.
 * Outputs: h_out device fp32 [B, d], the state after the last layer; with
 * w_unembed ([V, d] in cfg->dtype, V % 64 == 0 in bf16) and final_norm (fp32
 * [d]): logits_out (device fp32 [B, V], may be NULL) = W_unembed
 * RMSNorm(h; final_norm) (the normalised row rounded to bf16 in the bf16
 * path, fp32 accumulation) and next_out (device int32 [B], may be NULL) = the
 * arg max, ties to the lowest id.  w_unembed NULL: no head (V ignored).
 * Workspace: spider_decode_workspace_size(cfg, B, kv->cap, V) bytes (V = 0
 * without the head).
 * ------------------------------------------------------------------------ */
size_t spider_decode_workspace_size(const spider_decoder_cfg* cfg, int B, int cap, int V);

spider_status spider_decode_step(const spider_decoder_cfg* cfg, const spider_layer_weights* layers, int B,
                                 const int32_t* lens, const void* x, const spider_kv_cache* kv,
                                 const float* final_norm, const void* w_unembed, int V, float* h_out,
                                 float* logits_out, int32_t* next_out, void* workspace,
                                 size_t workspace_bytes, spider_stream stream);

/* ------------------------------------------------------------------------
 * spider_prefill_online - spider_prefill driven by the online skip
 * controller of ASL-Skip (Sec. 4.2.1, Eq. 4; Eq. 6 and Algorithm 1) instead
 * of a precomputed mask.  Sample b's last n_text rows are text, the rows
 * before them visual.  At every layer l < floor(L/2) (the decision window)
 * and for every visual row i not yet in skip mode, on the hidden state h
 * entering layer l:
 *   E_ii  = H(softmax(W_unembed h_i')) / ln V, the logit lens with no final
 *           norm; h_i' = bf16(h_i) in the bf16 path (the GEMM operand), h_i
 *           in fp32; H = natural-log Shannon entropy;
 *   F_itc = (1 + cos(h_i, q_b)) / 2, q_b = mean of sample b's text rows of h
 *           (cosine with a zero vector is 0);
 *   S_sa  = max(0, 1 - (E_ii + F_itc))                               (Eq. 4)
 *   acc_i += w1 * S_sa + w2 * slc_sel[l]  (double; acc starts at 0)
 *   acc_i >= T_skip: row i enters skip mode at layer l and bypasses
 *           sub-layer target[l] (0 attention, 1 FFN) in layers l .. L-1.
 * Layer l then runs (same semantics and precision as spider_prefill) with
 * the updated mask.  Text rows never skip.
 * Inputs as spider_prefill, plus: n_text >= 1 (every sample has at least
 *   n_text rows); w_unembed device [V, d] in cfg->dtype (16-byte aligned;
 *   bf16 needs V % 64 == 0); slc_sel HOST [L] doubles and target HOST [L]
 *   bytes as written by spider_slc_policy (entries l < floor(L/2) are read).
 * Outputs: codes_out HOST uint8 [L, rows], the mask the controller built
 *   (same encoding as spider_prefill's codes); admit_out HOST int32 [rows] or
 *   NULL: admission layer, -1 if never; s_sa_out device fp32
 *   [floor(L/2), rows] or NULL: S_sa of each row at each window layer where it
 *   was scored, 0 elsewhere; h_out as spider_prefill.
 * Synchronisation: with rows <= 256, B * n_text >= 5 and (bf16) fewer than
 *   128 heads x row blocks of 128 (ceil(rows / 128) * H < 128; with a bf16
 *   lens over V not a multiple of 128 also no 1..4 visual rows), the
 *   admissions, codes and row lists stay on the device and the launches of a
 *   window layer read the live row counts there; codes_out and admit_out are
 *   copied back once, after the last layer, and the call returns when the
 *   whole prefill has executed.  Otherwise the admission flags are read back
 *   to the host once per window layer (the call waits for the stream there)
 *   and the host builds the row lists: the call returns after the window has
 *   executed and the layers after it run asynchronously.  Both give the same
 *   h as spider_prefill on the returned codes, bit for bit.
 * Workspace: spider_prefill_online_workspace_size(cfg, B, rows, V) bytes.
 * ------------------------------------------------------------------------ */
size_t spider_prefill_online_workspace_size(const spider_decoder_cfg* cfg, int B, int rows, int V);

spider_status spider_prefill_online(const spider_decoder_cfg* cfg,
                                    const spider_layer_weights* layers, int B,
                                    const int32_t* cu_seqlens, const void* x, int n_text,
                                    const void* w_unembed, int V, const double* slc_sel,
                                    const uint8_t* target, double w1, double w2, double T_skip,
                                    uint8_t* codes_out, int32_t* admit_out, float* s_sa_out,
                                    float* h_out, void* workspace, size_t workspace_bytes,
                                    spider_stream stream);

/* ------------------------------------------------------------------------
 * spider_prefill_online_ablation - spider_prefill_online under the ablations
 * of the skip rule (Tab. 8 and its discussion; Sec. 4.2.1), selected by the
 * bits of `ablation` (0 gives spider_prefill_online exactly):
 *   SPIDER_ONLINE_NO_EII      the retention score is F_itc alone:
 *                             S_sa = max(0, 1 - F_itc);
 *   SPIDER_ONLINE_NO_FITC     the retention score is E_ii alone:
 *                             S_sa = max(0, 1 - E_ii);
 *   SPIDER_ONLINE_NO_ACCUM    no accumulation: acc_i = w1 * S_sa + w2 * slc_sel[l]
 *                             of the current window layer alone;
 *   SPIDER_ONLINE_WHOLE_LAYER without the SLC term: S_fuse = w1 * S_sa, and an
 *                             admitted row bypasses both sub-layers (code 3)
 *                             in layers l .. L-1 (target is then ignored but
 *                             must still be valid).
 * Arguments, outputs, workspace and synchronisation as spider_prefill_online;
 * bits outside these four give SPIDER_ERR_INVALID_ARG.  (The ablation without
 * S_sa, all visual rows following the offline SLC list, is spider_prefill with
 * a per-layer mask.)
 * ------------------------------------------------------------------------ */
#define SPIDER_ONLINE_NO_EII 1u
#define SPIDER_ONLINE_NO_FITC 2u
#define SPIDER_ONLINE_NO_ACCUM 4u
#define SPIDER_ONLINE_WHOLE_LAYER 8u

spider_status spider_prefill_online_ablation(const spider_decoder_cfg* cfg,
                                             const spider_layer_weights* layers, int B,
                                             const int32_t* cu_seqlens, const void* x, int n_text,
                                             const void* w_unembed, int V, const double* slc_sel,
                                             const uint8_t* target, double w1, double w2, double T_skip,
                                             uint32_t ablation, uint8_t* codes_out, int32_t* admit_out,
                                             float* s_sa_out, float* h_out, void* workspace,
                                             size_t workspace_bytes, spider_stream stream);

/* ------------------------------------------------------------------------
 * Kernel-class profiler (process-global, not thread-safe; for benchmarks).
 * When enabled, every launch of the library records a pair of HIP events on
 * its stream.  spider_profile_read() synchronises on the recorded events and
 * returns, for kernel class `cls` (0 .. spider_profile_classes()-1), the
 * number of launches and the summed kernel time in milliseconds since the
 * last reset.  spider_profile_enable(0) stops recording; (1) starts it and
 * resets the counters.  spider_profile_mask() restricts recording to the
 * classes whose bit is set (bit cls; all classes by default), so a timed
 * run can carry events around one kernel class only.
 * ------------------------------------------------------------------------ */
spider_status spider_profile_enable(int enable);
spider_status spider_profile_mask(uint32_t mask);
int spider_profile_classes(void);
const char* spider_profile_class_name(int cls);
spider_status spider_profile_read(int cls, int64_t* launches, double* total_ms);

#ifdef __cplusplus
}
#endif
#endif /* SPIDER_H */
