/*
 * echo.h -- C ABI of libecho, the MI355X (gfx950) implementation of the cached
 * DiT block step of EchoCache (energy-guided cross-modal caching for
 * audio-driven video generation).
 *
 * One step of the method, for one DiT block, is four calls:
 *
 *   echo_energy        audio -> per-latent-frame energy and weight
 *                      (Sec. 3.3, "Cross-modal Saliency Anchors"; once per clip)
 *   echo_select        per-token saliency = frame weight x relative change of the
 *                      block input against its cached input (Sec. 3.1 Eq. 1),
 *                      then top-K (or threshold) selection of tokens to recompute
 *                      (Sec. 3.3, saliency mask and k_t = ceil(N r_t))
 *   echo_block_partial the DiT block on the selected tokens only: queries from the
 *                      selected tokens, keys/values from all tokens, FFN on the
 *                      selected tokens (Sec. 3.3, "Fine-grained latent-level caching")
 *   echo_cache_update  int8 residual cache write for the selected tokens and
 *                      dequantized reuse for all others, fused into the block output
 *                      (Sec. 3.3 mask fusion; Sec. 3.4 reference + int8 residual)
 *
 * Conventions shared by every call
 *   - Tensor pointers are DEVICE pointers on the current HIP device, owned by
 *     the caller, row-major and 16-byte aligned.  The library allocates no
 *     memory: scratch space is a caller-provided workspace whose size the
 *     matching *_workspace() query returns.
 *   - Every call is asynchronous on `stream` (a hipStream_t passed as void*,
 *     NULL = the null stream) and never synchronises the host.
 *   - Arguments are validated before any HIP call; a rejected call launches
 *     nothing and writes nothing.  Errors are returned as echo_status codes;
 *     nothing throws across the ABI.  After ECHO_EDEVICE,
 *     echo_last_hip_error() returns the hipError_t of the failure (per thread).
 *   - Activation/weight storage is ECHO_F32 or ECHO_BF16 (bf16 = the upper 16
 *     bits of an IEEE fp32).  Accumulation is fp32 (fp64 where stated).
 *   - Token layout: L = T * N tokens, frame-major (token i is in latent frame
 *     floor(i / N)); one batch element.
 */
#ifndef ECHO_H
#define ECHO_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  ECHO_OK = 0,
  ECHO_EINVAL = 1,        /* null/misaligned pointer, size out of range, bad shape */
  ECHO_EUNSUPPORTED = 2,  /* well-formed but outside the supported shapes/dtypes   */
  ECHO_EWORKSPACE = 3,    /* workspace pointer null or smaller than required       */
  ECHO_EDEVICE = 4,       /* a HIP call failed; see echo_last_hip_error()          */
  ECHO_ELIMIT = 5         /* size above the fixed limit of an allocation-free call */
} echo_status;

typedef enum { ECHO_F32 = 0, ECHO_BF16 = 1 } echo_dtype;

/* Static string for a status code (never NULL). */
const char* echo_status_str(int status);
/* hipError_t of the last ECHO_EDEVICE on the calling thread (0 if none). */
int echo_last_hip_error(void);
/* Library version string, e.g. "0.1.0". */
const char* echo_version(void);

/* ------------------------------------------------------------------ energy */
/*
 * Audio energy anchor (Sec. 3.3, "Cross-modal Saliency Anchors").  The clip of
 * n_samples is split into T even segments, segment t = samples
 * [floor(t n / T), floor((t+1) n / T)); each segment gets an STFT (periodic
 * Hann window of n_fft, hop `hop`, no centring; a segment shorter than n_fft is
 * zero-padded to one frame; one-sided bins 0..n_fft/2).  Outputs (fp32):
 *   band_energy [T][n_bands]  sum of |X|^2 over the frames of segment t and the
 *                             bins of band b; bands have equal width on the mel
 *                             scale 2595 log10(1 + f/700) from 0 to sr/2
 *   frame_energy [T]          e_t = Frobenius norm of segment t's STFT
 *                             (= sqrt(sum_b band_energy[t][b]))
 *   frame_weight [T]          e_t / max_u e_u, or 1 for every t if all e are 0
 * Computed in fp64, rounded to fp32 once.  Requires 1 <= T <= 65535,
 * n_samples >= T, n_fft even in [16, 2048], 1 <= hop, 1 <= n_bands <= 64,
 * sample_rate > 0.  audio: device fp32 [n_samples].
 */
typedef struct {
  int32_t T;
  int32_t sample_rate;
  int32_t n_fft;
  int32_t hop;
  int32_t n_bands;
} echo_energy_cfg;

size_t echo_energy_workspace(const echo_energy_cfg* cfg, int64_t n_samples);
int echo_energy(const echo_energy_cfg* cfg, const float* audio, int64_t n_samples,
                float* band_energy, float* frame_energy, float* frame_weight,
                void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------ select */
/*
 * Saliency and recompute selection (Sec. 3.1 Eq. 1 per token; Sec. 3.3).
 *   delta_i = ||x_i - xref_i||_1 / (||xref_i||_1 + xi)   (fp64 sums)
 *   s_i     = fp32( fp64(frame_weight[floor(i / N)]) * delta_i )
 * Top-K mode (k >= 0): the k tokens first in the order (s descending, token
 * index ascending; a NaN s ranks above every number, -0 equals +0).
 * Threshold mode (k < 0): every token with s > threshold (or NaN s).
 * Outputs:
 *   idx [L] int32        the n_sel selected token indices, ascending, in
 *                        idx[0..n_sel); entries past n_sel are unspecified
 *   mask [L] uint8       1 for a selected token, 0 otherwise
 *   n_sel [1] int32      device scalar, the number selected (== k in top-K mode)
 *   saliency [L] fp32    s (optional, may be NULL)
 *   step_delta [1] fp64  sum_i num_i / (sum_i den_i + xi), the step-level Eq. 1
 *                        value against the cache (optional, may be NULL)
 * x, xref: [L][D] of `dtype`; frame_weight: fp32 [T].  Requires T, N >= 1,
 * L = T*N < 2^31, D >= 8 and D % 8 == 0, 0 <= k <= L or k < 0, xi >= 0.
 */
typedef struct {
  int32_t T;
  int32_t N;
  int32_t D;
  int32_t dtype;      /* echo_dtype of x and xref */
  int32_t k;          /* >= 0: top-k; < 0: threshold mode */
  float threshold;    /* threshold mode only */
  double xi;          /* Eq. 1 stabiliser, e.g. 1e-6 */
} echo_select_cfg;

size_t echo_select_workspace(const echo_select_cfg* cfg);
int echo_select(const echo_select_cfg* cfg, const void* x, const void* xref,
                const float* frame_weight, int32_t* idx, uint8_t* mask, int32_t* n_sel,
                float* saliency, double* step_delta,
                void* workspace, size_t workspace_bytes, void* stream);

/*
 * The two halves of echo_select, for callers that choose k from the step's
 * Eq. 1 value (the step schedule below): echo_saliency computes the saliency
 * (and, if step_delta is not NULL, the Eq. 1 value); echo_topk selects from a
 * given saliency with cfg->k / cfg->threshold as echo_select does.  Running
 * both gives exactly echo_select's results.  echo_saliency's workspace is
 * echo_saliency_workspace(cfg) bytes; echo_topk needs none.
 */
size_t echo_saliency_workspace(const echo_select_cfg* cfg);
int echo_saliency(const echo_select_cfg* cfg, const void* x, const void* xref,
                  const float* frame_weight, float* saliency, double* step_delta,
                  void* workspace, size_t workspace_bytes, void* stream);
int echo_topk(const echo_select_cfg* cfg, const float* saliency, int32_t* idx, uint8_t* mask,
              int32_t* n_sel, void* stream);

/*
 * echo_select without a workspace argument, for callers that cannot allocate
 * device memory: code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc.  Arguments, outputs and results are exactly those of
 * echo_select (bit-identical).  The scratch space echo_select takes from its
 * workspace (fp64 per-token sums; the fp32 saliency when `saliency` is NULL)
 * is instead a static device array of the library sized for
 * ECHO_SELECT_NOALLOC_MAX_TOKENS tokens (2.5 MiB); every GPU the library runs
 * on holds one copy of it until the process ends.  Its device address is
 * looked up on the first call on each device.  The call allocates nothing and
 * calls no hipMalloc or hipFree.  L = T*N above ECHO_SELECT_NOALLOC_MAX_TOKENS
 * returns ECHO_ELIMIT before anything is launched.  Every call on one GPU uses
 * that GPU's single array, and nothing in it needs to start at zero (each
 * call writes every entry it reads): calls that overlap on one GPU (other
 * streams, or threads without ordering between them) race for it and give
 * undefined results; calls ordered on one stream are safe.
 */
#define ECHO_SELECT_NOALLOC_MAX_TOKENS 131072
int echo_select_noalloc(const echo_select_cfg* cfg, const void* x, const void* xref,
                        const float* frame_weight, int32_t* idx, uint8_t* mask, int32_t* n_sel,
                        float* saliency, double* step_delta, void* stream);

/* ------------------------------------------------ two-stage selection */
/*
 * The literal form of the saliency anchors (Sec. 3.3, "Cross-modal Saliency
 * Anchors": top-k segments of the audio energy before generation; "Energy-
 * Guided Step-Latent Cache Scheduling": k_t = ceil(N r_t) latents per selected
 * segment) and the anchor strategies of the module ablation (Table 2:
 * Uniform, Random).
 *
 * echo_anchors writes anchors[T] (uint8 0/1):
 *   ECHO_ANCHOR_TOPK     the k segments ranked first by (keys desc, index asc),
 *                        NaN first.  keys [T] fp32: the frame energies of
 *                        echo_energy for the energy anchors, uniform random
 *                        numbers drawn by the caller for Random anchors;
 *   ECHO_ANCHOR_UNIFORM  the evenly spaced segments floor((2j + 1) T / (2k)),
 *                        j = 0..k-1 (keys unused, may be NULL).
 * Requires 1 <= T <= 4096, 0 <= k <= T.  One workgroup, O(T^2 / 1024) work.
 *
 * echo_topk_segments selects, in every anchor segment t (tokens [tN, tN + N)),
 * the min(k, N) tokens ranked first by (saliency desc, index asc), NaN first,
 * with the ranking rules of echo_topk; other segments' tokens are unselected.
 * Writes idx[0 .. n) ascending (n = number of anchors * min(k, N); idx must
 * hold that many, L always suffices), mask[L] (their indicator) and *n_sel = n
 * (device int32).  Give it the saliency of echo_saliency with unit frame
 * weights: a positive weight per segment cannot change the order inside one.
 * Requires 1 <= T <= 65535, N >= 1, T*N < 2^31, k >= 0.
 */
typedef enum { ECHO_ANCHOR_TOPK = 0, ECHO_ANCHOR_UNIFORM = 1 } echo_anchor_mode;

int echo_anchors(const float* keys, int32_t T, int32_t k, int32_t mode, uint8_t* anchors, void* stream);
int echo_topk_segments(const float* saliency, const uint8_t* anchors, int32_t T, int32_t N, int32_t k,
                       int32_t* idx, uint8_t* mask, int32_t* n_sel, void* stream);

/* ------------------------------------------------------------ token counts */
/*
 * Host functions (no device work) that fix how many tokens a step recomputes.
 *
 * echo_topk_count: K = ceil(ratio * L - 1e-9), clamped to [0, L] -- the
 * paper's k_t = ceil(N r_t) (Sec. 3.3, "Energy-Guided Step-Latent Cache
 * Scheduling") taken over all L tokens of the step (global top-K).  The
 * offset keeps products that are exact in decimal, such as 0.4 * 32760, from
 * rounding up through their binary representation.  Returns K, or
 * -ECHO_EINVAL for L < 1 or a ratio outside [0, 1] (NaN included).
 *
 * echo_segments_count: the number of tokens echo_topk_segments selects when
 * n_anchors segments of N tokens are anchors and k tokens are requested per
 * anchor segment: n_anchors * min(k, N).  Returns it, or -ECHO_EINVAL for
 * n_anchors < 0, N < 1, k < 0 or a count of 2^31 or more.
 */
int32_t echo_topk_count(double ratio, int32_t L);
int32_t echo_segments_count(int32_t n_anchors, int32_t N, int32_t k);

/* ---------------------------------------------------------- step schedule */
/*
 * Step-level cache schedule (Sec. 3.3, "Energy-Guided Step-Latent Cache
 * Scheduling"; Sec. 3.1 Eq. 2).  Host function: no device work.  Decides step
 * st->step and advances the state:
 *   step < n_full                     -> full step (k = L);
 *   otherwise acc += delta_t; if refresh_delta > 0 and acc > refresh_delta
 *                                     -> full step, acc = 0 (Eq. 2 refresh);
 *   otherwise dmax = max(dmax, delta_t); dhat = delta_t / dmax (0 if dmax == 0);
 *             r = clip(r_min + alpha * dhat, r_min, r_max);
 *             k = echo_topk_count(r, L).
 * delta_t is the step's Eq. 1 value (echo_saliency's step_delta); it is not
 * used on the leading full steps.  Returns k, or -ECHO_EINVAL for a bad
 * argument (L < 1, r_min > r_max, a rate outside [0, 1], NULL pointers).
 * *full is set to 1 for a full step, else 0.
 */
typedef struct {
  int32_t n_full;        /* leading full steps */
  double r_min;          /* minimum and maximum update ratio */
  double r_max;
  double alpha;          /* adjustment coefficient */
  double refresh_delta;  /* Eq. 2 threshold; <= 0: no refresh */
} echo_schedule_cfg;

typedef struct {
  int32_t step;          /* steps decided so far (start at 0) */
  double delta_max;      /* largest delta_t of the cached steps */
  double delta_acc;      /* delta_t accumulated since the last full step */
} echo_schedule_state;

int32_t echo_schedule_next(const echo_schedule_cfg* cfg, echo_schedule_state* st, double delta_t,
                           int32_t L, int32_t* full);

/* ------------------------------------------------------------ block partial */
/*
 * One adaLN DiT block on the selected tokens only (Sec. 3.3, "Fine-grained
 * latent-level caching": queries for the active tokens, keys and values from
 * the complete token set, attention on (Q', K, V), FFN on the active tokens):
 *   a    = LN(x) * (1 + scale1) + shift1                 all L rows
 *   q    = a[idx] Wq^T + bq ;  k = a Wk^T + bk ;  v = a Wv^T + bv
 *   o    = per-head softmax(q k^T / sqrt(D/H)) v          over all L keys
 *   x1   = x[idx] + gate1 * (o Wo^T + bo)
 *   y_sel= x1 + gate2 * (GELU_tanh(LN2(x1) W1^T + b1) W2^T + b2),
 *          LN2(z) = LN(z) * (1 + scale2) + shift2
 * LN: no affine, biased variance, eps = cfg->ln_eps.  Weights are [out][in]
 * (nn.Linear layout) in `dtype`: wq, wk, wv, wo [D][D]; w1 [F][D]; w2 [D][F];
 * biases bq, bk, bv, bo, b2 [D], b1 [F] in `dtype`; mod fp32 [6][D] = rows
 * shift1, scale1, gate1, shift2, scale2, gate2.
 * x [L][D] in `dtype`; idx [n_sel] int32 in [0, L) (any order, repeats allowed);
 * y_sel [n_sel][D] fp32, row j = output of token idx[j].  n_sel = 0 is a no-op.
 * Supported: ECHO_BF16 with D/H == 128, D % 256 == 0, F % 256 == 0 and
 * L*D, F*D, n_sel*F each below 2^30 elements (bf16 MFMA path; other shapes
 * return ECHO_EUNSUPPORTED); ECHO_F32 with D % 4 == 0, (D/H) % 4 == 0, D/H <= 128,
 * F % 4 == 0 (fp32 path for small shapes).  D <= 16384, F <= 65536.
 * Without ECHO_BLOCK_BATCH_INVARIANT the bf16 path splits the attention work
 * that does not fill a last round of the device along the keys (merged in
 * fp32), so a row's rounding may depend on how many rows are selected; the
 * result stays within the same tolerance of the definition either way.
 */
/* echo_block_cfg.flags */
#define ECHO_BLOCK_BATCH_INVARIANT 1 /* every token's y_sel row is bit-identical for
                                        any idx that contains the token (no work is
                                        split across workgroups by problem size) */

typedef struct {
  int32_t L;
  int32_t D;
  int32_t H;
  int32_t F;
  int32_t dtype;
  float ln_eps;
  int32_t flags;      /* 0 or ECHO_BLOCK_BATCH_INVARIANT; other bits: ECHO_EINVAL */
} echo_block_cfg;

typedef struct {
  const void* wq; const void* wk; const void* wv; const void* wo;
  const void* w1; const void* w2;
  const void* bq; const void* bk; const void* bv; const void* bo;
  const void* b1; const void* b2;
  const float* mod;
} echo_block_weights;

size_t echo_block_workspace(const echo_block_cfg* cfg, int32_t n_sel_max);
int echo_block_partial(const echo_block_cfg* cfg, const echo_block_weights* w,
                       const void* x, const int32_t* idx, int32_t n_sel, float* y_sel,
                       void* workspace, size_t workspace_bytes, void* stream);

/* -------------------------------------------------------- Wan-style block */
/*
 * The block of echo_block_partial with the extras of the Wan2.2-S2V family the
 * paper evaluates (Sec. 4), on the same restricted-query path (Sec. 3.3:
 * queries, cross-attention and FFN for the selected tokens; keys and values of
 * the self-attention from all tokens), for a batch of B elements that share
 * the weights (B = 2: the conditional and unconditional halves of
 * classifier-free guidance):
 *   a   = LN(x) * (1 + scale1) + shift1                          all rows
 *   q   = RoPE(RMSNorm(a[idx] Wq^T + bq) * gq)                   selected rows
 *   k   = RoPE(RMSNorm(a Wk^T + bk) * gk);  v = a Wv^T + bv      all rows
 *   x1  = x[idx] + gate1 * (attn(q, k, v) Wo^T + bo)
 *   c   = LN(x1) * g3 + b3
 *   qc  = RMSNorm(c Wqc^T + bqc) * gqc
 *   kc  = RMSNorm(ctx Wkc^T + bkc) * gkc;  vc = ctx Wvc^T + bvc  all context rows
 *   x2  = x1 + attn(qc, kc, vc) Woc^T + boc
 *   y_sel = x2 + gate2 * (GELU_tanh(LN2(x2) W1^T + b1) W2^T + b2)
 * RMSNorm(z) = z / sqrt(mean(z^2) + rms_eps) over all D channels.  RoPE: token
 * i of the T x gh x gw latent grid sits at (t, r, c) = (i / (gh gw),
 * (i / gw) % gh, i % gw); the dh/2 channel pairs (2j, 2j+1) of every head turn
 * by t, r and c times base^(-j'/n) for the first dh/2 - 2(dh/6) pairs, the
 * next dh/6 and the last dh/6 respectively (j' and n: the pair's index within
 * its axis and the axis's pair count).  Attention as in echo_block_partial;
 * the self-attention of element b sees the keys of element b only, the
 * cross-attention the Lc context rows of element b.
 * x [B][L][D] and ctx [B][Lc][D] in `dtype`; idx [sum n_sel] device int32:
 * global rows b * L + i, element by element (the rows of element b are
 * idx[o_b .. o_b + n_sel[b]) with o_b = n_sel[0] + .. + n_sel[b-1]), any order
 * within an element; n_sel is a HOST array of B counts; y_sel [sum n_sel][D]
 * fp32 in idx order.  Weights as in echo_block_weights, the cross-attention
 * matrices [D][D] and biases [D] in `dtype`; gq, gk, gqc, gkc, g3, b3 fp32 [D].
 * Supported: ECHO_BF16 with D/H == 128, D % 256 == 0, F % 256 == 0, T*gh*gw ==
 * L, and B*L*D, B*Lc*D, sum(n_sel)*F each below 2^30 elements.
 */
typedef struct {
  int32_t B;
  int32_t L;
  int32_t D;
  int32_t H;
  int32_t F;
  int32_t Lc;          /* context rows per element */
  int32_t T, gh, gw;   /* latent grid, T * gh * gw == L */
  int32_t dtype;
  float ln_eps;
  float rms_eps;
  double rope_base;    /* e.g. 10000 */
  int32_t flags;       /* 0 or ECHO_BLOCK_BATCH_INVARIANT */
} echo_wan_block_cfg;

typedef struct {
  echo_block_weights self;            /* modulation, self-attention and FFN */
  const void* wqc; const void* wkc; const void* wvc; const void* woc;
  const void* bqc; const void* bkc; const void* bvc; const void* boc;
  const float* gq; const float* gk;   /* self-attention RMSNorm weights */
  const float* gqc; const float* gkc; /* cross-attention RMSNorm weights */
  const float* g3; const float* b3;   /* cross-attention LN scale and shift */
} echo_wan_block_weights;

size_t echo_wan_block_workspace(const echo_wan_block_cfg* cfg, int32_t n_total_max);
int echo_wan_block_partial(const echo_wan_block_cfg* cfg, const echo_wan_block_weights* w, const void* x,
                           const void* ctx, const int32_t* idx, const int32_t* n_sel, float* y_sel,
                           void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------- cache update */
/*
 * Cache write and mask fusion (Sec. 3.3: out = m * fresh + (1 - m) * cached;
 * Sec. 3.4: cached output = reference + dequantized int8 residual, converted
 * back to the compute precision).  One reference per token, xref_i = the block
 * input at its last recompute.  For each selected row i = idx[j]:
 *   res = fp32(y_sel[j] - x_i); amax = max|res|;
 *   scale_i = fp32(amax / 127); code = clamp(rint(fp32(res * fp32(127 / amax))), +-127)
 *   (amax == 0 -> scale 0, codes 0); xref_i = x_i; y_i = cast(y_sel[j])
 * For each unselected row (mask == 0): y_i = cast(fp32(xref_i + fp32(scale_i * code)))
 * cast = round to nearest even into `dtype`.  x, xref, y: [L][D] `dtype`;
 * codes [L][D] int8; scale [L] fp32; xref, codes and scale are updated in place.
 * idx must hold n_sel distinct rows and mask must be their indicator.
 * Requires D % 8 == 0, D <= 16384.
 */
typedef struct {
  int32_t L;
  int32_t D;
  int32_t dtype;
} echo_cache_cfg;

int echo_cache_update(const echo_cache_cfg* cfg, const void* x, const int32_t* idx,
                      const uint8_t* mask, int32_t n_sel, const float* y_sel,
                      void* xref, int8_t* codes, float* scale, void* y, void* stream);

/*
 * The cache codecs of the module ablation (Table 2: "FP16" and "Naive INT8"
 * against the residual int8 cache), with echo_cache_update's fusion:
 *   ECHO_CODEC_RESIDUAL_INT8  exactly echo_cache_update (store unused, may be NULL);
 *   ECHO_CODEC_FULL           a selected row stores cast(y_sel[j]) into store_i;
 *                             an unselected row outputs store_i unchanged
 *                             (store [L][D] `dtype`; codes and scale unused,
 *                             may be NULL);
 *   ECHO_CODEC_NAIVE_INT8     a selected row is quantized itself: amax = max|y_sel[j]|,
 *                             scale and codes as above with res = y_sel[j];
 *                             an unselected row outputs cast(fp32(scale_i * code))
 *                             (store unused, may be NULL).
 * Every codec sets xref_i = x_i and y_i = cast(y_sel[j]) for a selected row.
 * Requirements as for echo_cache_update.
 */
typedef enum {
  ECHO_CODEC_RESIDUAL_INT8 = 0,
  ECHO_CODEC_FULL = 1,
  ECHO_CODEC_NAIVE_INT8 = 2
} echo_codec;

int echo_cache_update_codec(const echo_cache_cfg* cfg, int32_t codec, const void* x, const int32_t* idx,
                            const uint8_t* mask, int32_t n_sel, const float* y_sel, void* xref, void* store,
                            int8_t* codes, float* scale, void* y, void* stream);

/* ---------------------------------------------- adaptive reference cache */
/*
 * The paper's memory-efficient cache (Sec. 3.4, "Memory-efficient Cache
 * Management") in place of echo_cache_update's one-reference-per-token form:
 * a fresh output y whose cosine similarity <y, r> / (|y| |r|) with its chain's
 * current reference r exceeds tau is kept as an int8 residual against r
 * (res = fp32(y - r), codes and scale as in echo_cache_update); otherwise y
 * itself is stored in `dtype` and becomes the chain's current reference.  A
 * chain is chain_len consecutive tokens (one spatial row of the latent grid)
 * and keeps its current reference across updates; the similarity is taken in
 * fp64 (0 if a norm is 0) and compared strictly.  Before the write, the old
 * entries of the rewritten tokens are dropped; a reference that no entry and
 * no chain holds any more is released to the free slots.
 *
 * Fusion: selected row i = idx[j] outputs cast(y_sel[j]) and records
 * xref_i = x_i (the saliency reference of echo_select); an unselected row
 * outputs its reference row, or cast(fp32(r + fp32(scale_i * code))) for a
 * residual entry, or zeros if it never had an entry.
 *
 * State: caller-owned device arrays (echo_refcache_state), prepared once by
 * echo_refcache_init.  capacity >= L + L / chain_len reference slots always
 * suffice (every live slot is held by an entry or a chain).  The number of
 * live references is capacity - *free_top.  x, xref, y: [L][D] `dtype`;
 * idx [n_sel] ascending distinct rows with mask their indicator; y_sel
 * [n_sel][D] fp32.  Requires L % chain_len == 0, D % 8 == 0, D <= 16384, tau
 * finite.  Slot numbers depend on the order of atomic operations; stored
 * values, decisions and outputs do not.
 */
typedef struct {
  int32_t L;
  int32_t D;
  int32_t dtype;
  int32_t chain_len;
  int32_t capacity;
  float tau;
} echo_refcache_cfg;

typedef struct {
  void* pool;          /* [capacity][D] `dtype`: reference rows */
  int32_t* refcount;   /* [capacity] holders of each slot */
  int32_t* free_list;  /* [capacity] stack of free slots */
  int32_t* free_top;   /* [1] number of free slots */
  int32_t* chain_ref;  /* [L / chain_len] current reference slot, -1 = none */
  int32_t* ent_slot;   /* [L] slot of the token's entry, -1 = none */
  uint8_t* ent_kind;   /* [L] 0 none, 1 reference, 2 residual */
  int8_t* codes;       /* [L][D] residual codes */
  float* scale;        /* [L] residual scales */
} echo_refcache_state;

int echo_refcache_init(const echo_refcache_cfg* cfg, const echo_refcache_state* st, void* stream);
int echo_refcache_update(const echo_refcache_cfg* cfg, const echo_refcache_state* st, const void* x,
                         const int32_t* idx, const uint8_t* mask, int32_t n_sel,
                         const float* y_sel, void* xref, void* y, void* stream);

/* ------------------------------------------------------------ kernel timing */
/*
 * Optional per-kernel timing with HIP events, for the calling thread.
 * echo_profile_enable(1) makes every later launch record a start/stop event
 * pair on its stream; echo_profile_read() waits for the recorded events, fills
 * up to `max` entries (kernel name, number of launches, summed milliseconds)
 * and clears the record.  Returns the number of entries written, or a negative
 * echo_status on failure.  Enabling adds two event records per launch.
 */
typedef struct {
  const char* name;
  int64_t launches;
  double total_ms;
} echo_kernel_time;

int echo_profile_enable(int on);
int echo_profile_read(echo_kernel_time* out, int32_t max);

/* ------------------------------------------------------ sustained MFMA rate */
/*
 * Diagnostic for the measurement of the matrix kernels, not part of the
 * cached step.  The nominal bf16 peak (2516.6 TFLOP/s on a 256-CU part at
 * 2.4 GHz) assumes the clock holds while the matrix cores work; it holds only
 * while they switch few bits.  echo_mfma_ceiling runs a dense bf16 MFMA
 * instruction stream with nothing else in its loop for `seconds` (after a
 * warm-up of a third of that) and writes the sustained rate in TFLOP/s to
 * *tflops: the ceiling the path's matrix kernels can reach on the same data.
 *   pattern ECHO_MFMA_ATTENTION: 12 waves per CU, v_mfma_f32_32x32x16_bf16,
 *           a new LDS operand for every MFMA (the attention's S and PV);
 *   pattern ECHO_MFMA_GEMM: 4 waves per CU, 8 x 8 grids of
 *           v_mfma_f32_16x16x32_bf16 tiles, 16 LDS fragment reads per 64
 *           MFMAs (the four-wave GEMM without its global-to-LDS copies);
 *   data ECHO_OPERANDS_CONSTANT: operands 1 + j/8;
 *   data ECHO_OPERANDS_GAUSSIAN: A ~ N(0, 1), B ~ N(0, 0.02) rounded to bf16
 *        (the path's activations and weights).
 * Synchronous on `stream`; allocates a small result buffer on it.  Returns
 * ECHO_EINVAL for an unknown pattern or data kind, seconds outside (0, 60]
 * or a null tflops, ECHO_EDEVICE on a HIP error.
 */
typedef enum { ECHO_MFMA_ATTENTION = 0, ECHO_MFMA_GEMM = 1 } echo_mfma_pattern;
typedef enum { ECHO_OPERANDS_CONSTANT = 0, ECHO_OPERANDS_GAUSSIAN = 1 } echo_operand_data;

int echo_mfma_ceiling(int32_t pattern, int32_t data, double seconds, double* tflops, void* stream);

#ifdef __cplusplus
}
#endif
#endif /* ECHO_H */
