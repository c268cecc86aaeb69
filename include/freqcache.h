/*
 * freqcache.h -- C ABI of the FreqCache per-step hot path on AMD Instinct MI355X (gfx950).
 *
 * FreqCache (arXiv 2604.24391) decides, at every navigation step, which visual
 * tokens of the current camera frame may reuse cached model results, and the
 * model then recomputes only the others.  This library implements that step:
 *
 *   fc_select        frequency-guided cacheable-token selection (Sec. 4.1-4.4,
 *                    Algorithm 1): per-patch DFT amplitude spectra of both
 *                    frames, global spectral similarity and migration gate,
 *                    phase-correlation displacement and alignment mask,
 *                    block-DCT high-frequency energy and refresh mask,
 *                    spectral-entropy reuse budget, ascending-energy top-K.
 *   fc_cache_update  token-cache preparation for the new step: each reused
 *                    token takes the cached rows of its aligned source token
 *                    in the previous frame (Sec. 4.1, Eq. 4-2).
 *   fc_layer_forward the partial-recompute decoder layer: only non-reused
 *                    tokens are gathered through RMSNorm, QKV, attention over
 *                    the full cached K/V, O-projection and the SwiGLU MLP, and
 *                    scattered back into the token cache (Sec. 1, 2.2, 5.2).
 *
 * Conventions for every call:
 *   - Pointers are DEVICE pointers unless marked (host).  The caller allocates
 *     and owns every buffer; the library never frees or keeps caller pointers
 *     past the call.  A context owns only its workspace and constant tables,
 *     sized once by fc_create, so no call allocates device memory.
 *   - Work is enqueued asynchronously on `stream` (a hipStream_t; NULL = the
 *     default stream); results are valid once the stream reaches the call.
 *     Nothing is read back to the host: counts produced by fc_select stay on
 *     the device and fc_layer_forward reads them there.
 *   - Argument and shape checks are synchronous and launch nothing.  Every call
 *     returns an fc_status; on failure fc_last_error() describes it.  A launch
 *     failure returns FC_ERR_HIP.  The library never aborts or exits.
 *   - Identical inputs give byte-identical outputs (no floating-point atomics).
 *   - A context must not be used from two host threads at once; calls on one
 *     context that overlap on different streams race on its workspace.
 *   - bf16 values are raw uint16_t bit patterns.  Matrices are row-major;
 *     weights are [out][in] like torch.nn.Linear.
 */
#ifndef FREQCACHE_H
#define FREQCACHE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct fc_ctx fc_ctx;

typedef enum {
  FC_OK = 0,
  FC_ERR_INVALID_ARG = 1,   /* null pointer, out-of-range parameter        */
  FC_ERR_SHAPE = 2,         /* sizes inconsistent with each other           */
  FC_ERR_CAPACITY = 3,      /* sizes above what the context was created for */
  FC_ERR_HIP = 4,           /* a HIP runtime call or kernel launch failed   */
  FC_ERR_NO_DEVICE = 5,     /* no usable GPU                                */
  FC_ERR_UNSUPPORTED = 6    /* a valid request the library does not handle  */
} fc_status;

/* Upper bounds fixed at context creation; they size the workspace.  (host) */
typedef struct {
  int32_t max_batch;        /* frame pairs / episodes per call                    */
  int32_t max_height;       /* frame height in pixels                             */
  int32_t max_width;        /* frame width in pixels                              */
  int32_t max_tokens;       /* visual tokens per frame N (<= 1024)                */
  int32_t max_seq;          /* cached sequence length S = T + W * N               */
  int32_t max_d_model;      /* hidden size                                        */
  int32_t max_ffn;          /* SwiGLU intermediate size                           */
  int32_t max_qkv;          /* (n_heads + 2 n_kv_heads) * head_dim                */
} fc_caps;

/* Selection hyper-parameters.  (host; copied at call time)
 * Defaults from the paper (Sec. 6.4): tau_mig 0.12, lambda 0.25, alpha_min 0.08,
 * alpha_max 0.5. */
typedef struct {
  int32_t patch;            /* P, pixels per patch side (14); 2..32                         */
  int32_t merge;            /* m, patches per token side (1 or 2)                           */
  double tau_mig;           /* flush when Sim_freq < tau_mig (Sec. 4.1)                    */
  double lambda_;           /* refresh when E > mu_E + lambda sigma_E (Eq. 4-3)            */
  double alpha_min;         /* reuse-ratio bounds of Eq. 4-4                               */
  double alpha_max;
  int32_t adaptive;         /* 1: alpha from spectral entropy (Eq. 4-4); 0: alpha_fixed    */
  double alpha_fixed;       /* fixed reuse ratio (the "w/o Module III" ablation, Table 3)  */
  int32_t entropy_norm;     /* 1: entropy divided by ln(grid bins), so Psi is in [0, 1]    */
  double tau_sim;           /* extra per-token similarity floor; 0 = exact Algorithm 1     */
  /* Module ablations of Table 3 (Sec. 6.3); 0 (zero-initialised) = the full method.       */
  int32_t no_align;         /* 1: "w/o Module I", position-wise matching: shift = (0, 0)
                               and every token aligned (phase correlation not used)       */
  int32_t no_refresh;       /* 1: "w/o Module II", no token is refreshed by its edge energy
                               (mu_E, sigma_E and the threshold are still reported)       */
  /* The paper's naive frequency baseline (Sec. 6.1: position-wise amplitude similarity,
     static reuse above a fixed threshold tau) is no_align = 1, no_refresh = 1,
     adaptive = 0 with alpha_fixed = 1, tau_mig = 0 and tau_sim = tau.                     */
  int32_t align_pixel;      /* 1: Module I's displacement from Eq. 4-1 on the full-resolution
                               luma (fc_phase_correlate), rounded to whole tokens of P m
                               pixels (halves away from zero), instead of the token-grid map.
                               Needs H and W of the form 7 * 2^k (14 ... 896); the first such
                               call on a context allocates its workspace.  fc_select and
                               fc_select_noalloc only (not fc_select_carry).               */
  int32_t align_rotation;   /* with align_pixel = 1: the rotation of the current frame is found
                               first and undone (fc_phase_correlate_rotation), and the token
                               displacement is that of the frame centre.  Needs
                               min(H, W) >= 28.                                             */
} fc_select_params;

enum { FC_SCALAR_SIM_FREQ = 0, FC_SCALAR_PSI, FC_SCALAR_ALPHA, FC_SCALAR_MU,
       FC_SCALAR_SIGMA, FC_SCALAR_THR, FC_NSCALARS };
enum { FC_COUNT_K_REUSE = 0, FC_COUNT_K_CAND, FC_COUNT_K_FINAL, FC_COUNT_FLUSHED,
       FC_NCOUNTS };
enum { FC_FLAG_ALIGNED = 1, FC_FLAG_FRESH = 2, FC_FLAG_CAND = 4 };

/* Outputs of fc_select; caller-allocated device buffers.  N = tokens per frame
 * = (H / (P m)) * (W / (P m)); token ids are row-major on the token grid. */
typedef struct {
  float *sim;               /* [B][N] aligned per-token spectral similarity (Eq. 3-3 per token; 0 if unaligned) */
  double *energy;           /* [B][N] token high-frequency energy (Eqs. 3-4/3-5; sum over the m*m patches)      */
  uint8_t *reuse_mask;      /* [B][N] 1 = the token reuses its cached results (P_final of Algorithm 1)          */
  int32_t *recompute_idx;   /* [B][N] ascending ids of recomputed tokens; the first n_recompute[b] are valid    */
  int32_t *n_recompute;     /* [B]    N - K_final                                                               */
  int32_t *shift;           /* [B][2] (di, dj): token (I, J) reuses source token (I + di, J + dj) (Eq. 4-1)     */
  double *scalars;          /* [B][FC_NSCALARS] Sim_freq, Psi, alpha_t, mu_E, sigma_E, mu_E + lambda sigma_E    */
  int32_t *counts;          /* [B][FC_NCOUNTS] K_reuse, K_candidate, K_final, flushed                          */
  uint8_t *flags;           /* [B][N] optional (may be NULL): FC_FLAG_* bits of Mask_align, Mask_fresh, C       */
} fc_select_out;

/* One decoder block (pre-norm RMSNorm, q/k/v bias, rotate-half RoPE, GQA, SwiGLU).
 * (host struct; the weight pointers are device pointers, bf16) */
typedef struct {
  int32_t d_model, n_heads, n_kv_heads, head_dim, d_ffn;
  float rms_eps;            /* 1e-6 */
  double rope_theta;        /* 1e6  */
  const uint16_t *w_qkv;    /* [(n_heads + 2 n_kv_heads) head_dim][d_model], rows q | k | v */
  const uint16_t *b_qkv;    /* [(n_heads + 2 n_kv_heads) head_dim]                          */
  const uint16_t *w_o;      /* [d_model][n_heads head_dim]                                  */
  const uint16_t *w_gate;   /* [d_ffn][d_model]                                             */
  const uint16_t *w_up;     /* [d_ffn][d_model]                                             */
  const uint16_t *w_down;   /* [d_model][d_ffn]                                             */
  const uint16_t *g_attn;   /* [d_model] RMSNorm gain before attention                      */
  const uint16_t *g_mlp;    /* [d_model] RMSNorm gain before the MLP                        */
} fc_layer_desc;

/* One layer's token cache.  Sequence layout: [T text tokens][W frame slots of N
 * tokens][U text tokens].  The frame slots are a ring: physical slot p holds the frame with
 * logical index (p - head) mod W (0 = oldest, W - 1 = current).  A key sits at
 * position T + logical * N + token (text: its index), i.e. at its place in the
 * current step's prompt.  K holds raw (pre-RoPE) keys; rotation happens on use,
 * so advancing the window (head = (head + 1) mod W) moves no data.  (host struct) */
typedef struct {
  uint16_t *k;              /* [B][S][n_kv_heads][head_dim] bf16, S = T + W N */
  uint16_t *v;              /* [B][S][n_kv_heads][head_dim] bf16              */
  int32_t text_tokens;      /* T */
  int32_t frame_tokens;     /* N */
  int32_t window;           /* W >= 1 (frames kept, including the current one) */
  int32_t head;             /* 0 <= head < W */
  /* Multimodal RoPE of Qwen2.5-VL (all zero: 1-D RoPE by prompt index).  The rotary
     frequency pairs are split into sections of mrope_section[0..2] pairs (sum
     head_dim / 2, each a multiple of 8) rotated by a token's temporal, row and column
     position: text token p has (p, p, p); token (I, J) of the frame with logical index l
     (0 = oldest) has (st, st + I, st + J), st = T + l max(N / grid_w, grid_w).  Causality
     stays by prompt index. */
  int32_t grid_w;           /* token-grid width of a frame (M-RoPE only)      */
  int32_t mrope_section[3];
  /* Text after the frames: U tokens at rows (and prompt indices) T + W N + u, e.g. the
     instruction that follows the current image.  They come after the current frame,
     so fc_layer_forward_trail recomputes all of them at every step; frame tokens never
     attend to them.  With M-RoPE their three positions are T + W span + u.  0: none. */
  int32_t trail_tokens;
  /* Slot map (NULL: every row is stored at its own index).  Otherwise the first part of
     a slot state of fc_slot_state_bytes(B, S) bytes (device, int32), set up by
     fc_slot_map_init: row r of item b lives at pool row slot_map[b S + r] of the same
     K and V arrays.  One state serves every layer of the item (all layers share the
     reuse decisions), so all layers' caches point at the same state.  A reused token
     then shares its source's pool row: fc_cache_update_layers moves no K/V bytes, it
     updates the map (reference-counted pool rows, freed when no row maps to them). */
  int32_t *slot_map;
} fc_kv_cache;

/* One vision-encoder block (Qwen2.5-VL style; host struct, device bf16 pointers):
 * pre-norm RMSNorm, q/k/v with bias, 2-D rotary positions, bidirectional attention,
 * output projection with bias, SiLU-gated MLP with biases.
 *   w_qkv [3 d][d] (rows q | k | v, each head's head_dim dims contiguous), b_qkv [3 d];
 *   w_o [d][d], b_o [d]; w_gate_up [2 d_ffn][d] (gate rows, then up rows),
 *   b_gate_up [2 d_ffn]; w_down [d][d_ffn], b_down [d]; g1, g2 [d] RMSNorm gains.
 * d = n_heads head_dim; d and d_ffn multiples of 64 (pad the MLP with zero rows,
 * columns and biases: exact); head_dim a multiple of 16 up to 128. */
typedef struct {
  int32_t d_model, n_heads, head_dim, d_ffn;
  float rms_eps;            /* 1e-6 */
  double rope_theta;        /* 1e4: frequencies theta^(-2 i / (head_dim / 2)), i < head_dim / 4 */
  const uint16_t *w_qkv, *b_qkv, *w_o, *b_o, *w_gate_up, *b_gate_up, *w_down, *b_down;
  const uint16_t *g1, *g2;
} fc_vit_desc;

/* The encoder's per-layer cache of one frame: raw (pre-rotary) keys and values of every
 * patch, patches token-major: the merge x merge patches of merged token t = (I, J) are
 * rows t merge^2 + a merge + c, at patch-grid position (I merge + a, J merge + c).
 *   k, v: [B][grid_h grid_w merge^2][n_heads][head_dim] bf16 (device). */
typedef struct {
  uint16_t *k, *v;
  int32_t grid_h, grid_w;   /* merged-token grid of the frame */
  int32_t merge;            /* patches per merged token side (1 to 4; Qwen2.5-VL: 2) */
  int32_t window;           /* attention window side in merged tokens (Qwen2.5-VL: 4,
                               i.e. 112 px at 14-px patches and 2 x 2 merge); 0 = full
                               attention over the frame */
  /* fc_vit_cache_update only: NULL, NULL = k, v hold the previous frame and are remapped
     in place (the frame's old rows staged first); otherwise the previous frame's k, v
     (same layout, buffers overlapping neither k nor v), from which the reused rows are
     copied into k, v
     (callers alternate two caches per block; no staging) */
  const uint16_t *k_prev, *v_prev;
} fc_vit_cache;

/* The encoder's patch merger (Qwen2.5-VL style; host struct, device bf16 pointers): each
 * patch row RMS-normalised (gain g), the merge^2 patch rows of a merged token
 * concatenated (hidden = merge^2 d_model), then hidden -> hidden with bias, exact (erf)
 * GELU, hidden -> d_out with bias.
 *   g [d_model]; w1 [hidden][hidden], b1 [hidden]; w2 [d_out][hidden], b2 [d_out].
 * d_model a multiple of 64 up to 2048; d_out a multiple of 16. */
typedef struct {
  int32_t d_model, merge, d_out;
  float rms_eps;            /* 1e-6 */
  const uint16_t *g, *w1, *b1, *w2, *b2;
} fc_merger_desc;

/* Library version string. */
const char *fc_version(void);

/* Text of the last non-OK status returned on this host thread ("" if none). */
const char *fc_last_error(void);

/* Create a context on `device`, sizing its workspace for `caps` (host).
 * Returns FC_ERR_NO_DEVICE when no GPU is visible. */
fc_status fc_create(fc_ctx **out, int32_t device, const fc_caps *caps);
fc_status fc_destroy(fc_ctx *ctx);

/* Cacheable-token selection for B frame pairs (Algorithm 1 per pair).
 *   frames_prev: [B][3][H][W] float32 RGB in [0, 1], or NULL (no previous frame:
 *                treated as an all-zero frame, so the step is flushed, Sec. 4.1);
 *   frames_cur:  [B][3][H][W] float32.
 * H and W must be multiples of P m; N = (H/(P m)) (W/(P m)) <= 1024 and <= caps.
 * Every field of `out` except `flags` must be non-NULL. */
fc_status fc_select(fc_ctx *ctx, const fc_select_params *prm, const float *frames_prev,
                    const float *frames_cur, int32_t B, int32_t H, int32_t W,
                    const fc_select_out *out, void *stream);

/* Bytes of the carried selection state of a batch of B frames of H x W pixels (the
 * spectra of one frame per item: per-patch DFT amplitudes and mean luma; an opaque
 * device buffer the caller allocates, at least 16-byte aligned).  0 for sizes that
 * hold no patch.  (host function, no device work) */
size_t fc_select_state_bytes(int32_t B, int32_t H, int32_t W);

/* fc_select along an episode, with the previous frame's spectra carried from the
 * previous step instead of recomputed from its pixels (Algorithm 1 needs the
 * previous frame only through its per-patch amplitude spectra and patch means).
 *   state_prev: the state_cur of the previous call on the same frame size and batch,
 *               or NULL at the first step (no previous frame: flushed, as fc_select
 *               with frames_prev = NULL);
 *   state_cur:  receives this frame's spectra; fc_select_state_bytes(B, H, W) bytes,
 *               not overlapping state_prev (callers alternate two buffers).
 * Outputs are byte-identical to fc_select on the pixels of both frames.  The states
 * hold no meaning for other sizes or parameters of P (not checked). */
fc_status fc_select_carry(fc_ctx *ctx, const fc_select_params *prm, const void *state_prev,
                          const float *frames_cur, void *state_cur, int32_t B, int32_t H,
                          int32_t W, const fc_select_out *out, void *stream);

/* fc_select without a context and without any device allocation, for callers that
 * cannot allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc).  Same arguments, kernels and outputs as fc_select,
 * on the calling thread's current device; the workspace (per-patch amplitudes, means,
 * energies and spectral products: about 0.85 MB per 448x448 pair) lives in a static
 * device array of 16 MiB that each GPU holds until the process ends.
 *   - Sizes whose workspace exceeds 16 MiB return FC_ERR_CAPACITY before any device
 *     work (e.g. at most 19 pairs of 448x448 frames, 4 of 896x896).
 *   - The first call on a device does a one-time set-up that synchronises with it
 *     (architecture check, the array's device address, the transform tables); make
 *     that first call outside graph capture.  Later calls only launch kernels.
 *   - Every call on one GPU shares that GPU's array: calls that overlap in time on
 *     one GPU (other streams, other host threads) race and must be serialised by the
 *     caller.  Nothing in the array needs clearing between calls. */
fc_status fc_select_noalloc(const fc_select_params *prm, const float *frames_prev,
                            const float *frames_cur, int32_t B, int32_t H, int32_t W,
                            const fc_select_out *out, void *stream);

/* The text rows after the frames (kv->trail_tokens = U > 0) through the same decoder
 * block, all U of them, after fc_layer_forward of this layer at this step (their
 * queries attend to the whole cache, the current frame's new rows included):
 *   x_trail: [B][U][d_model] bf16 layer input of the trailing text;
 *   y_trail: [B][U][d_model] bf16 output; the K/V rows T + W N + u are written. */
fc_status fc_layer_forward_trail(fc_ctx *ctx, const fc_layer_desc *layer, const fc_kv_cache *kv,
                                 const uint16_t *x_trail, uint16_t *y_trail, int32_t B,
                                 void *stream);

/* Token-cache preparation for one layer at a new step.  The caller has already
 * advanced kv->head, so the current frame lives in slot (head + W - 1) mod W and
 * the previous frame in slot (head + W - 2) mod W (the same slot when W = 1).  For
 * every token t with reuse_mask[b][t] = 1, the K/V rows of the current slot and
 * y_cur[b][t] are copied from source token s = (I + di) grid_w + (J + dj) of the
 * previous frame (K/V) and of y_prev.  Other rows are left untouched (the layer
 * call rewrites them).
 *   y_prev, y_cur: [B][N][d_model] bf16, non-overlapping (else FC_ERR_INVALID_ARG);
 *   shift [B][2], reuse_mask [B][N]: from fc_select; grid_w: token-grid width. */
fc_status fc_cache_update(fc_ctx *ctx, const fc_layer_desc *layer, const fc_kv_cache *kv,
                          const uint16_t *y_prev, uint16_t *y_cur, const int32_t *shift,
                          const uint8_t *reuse_mask, int32_t grid_w, int32_t B, void *stream);

/* The same remap as fc_cache_update for the caches of n_layers layers at once (Sec. 4.1 /
 * Eq. 4-2): kvs[l], y_prev[l] and y_cur[l] (host arrays of n_layers entries, device
 * pointers inside) are layer l's cache and output buffers.  The layers share `layer`'s
 * dimensions and the caches' text_tokens, frame_tokens, window, head and trail_tokens
 * (all advanced to the same step); otherwise FC_ERR_SHAPE.  No two layers' K, V or
 * output buffers may overlap: the layers are copied concurrently (checked for the output
 * buffers: a y_cur overlapping any y_prev or another layer's y_cur is FC_ERR_INVALID_ARG).
 *   y_prev, y_cur: both NULL moves no output rows (the layer calls read only the
 *     recomputed rows of their inputs; skip them when the reused tokens' outputs are
 *     not consumed), else as in fc_cache_update.
 *   Slot-mapped caches (every kvs[l].slot_map the same state, else FC_ERR_INVALID_ARG):
 *     no K/V row moves; the map of each item is updated once for all layers: the rows
 *     of the frame that left the window release their pool rows, each reused token
 *     maps to its source's pool row, each recomputed token takes a free pool row.
 *   Otherwise equivalent to fc_cache_update on each layer in turn (a window of one frame,
 *     an in-place overwrite, runs those per-layer calls). */
fc_status fc_cache_update_layers(fc_ctx *ctx, const fc_layer_desc *layer, int32_t n_layers,
                                 const fc_kv_cache *kvs, const uint16_t *const *y_prev,
                                 uint16_t *const *y_cur, const int32_t *shift,
                                 const uint8_t *reuse_mask, int32_t grid_w, int32_t B,
                                 void *stream);

/* Bytes of the slot state of B items with S cache rows (S = T + W N + U): the map
 * [B][S] (the slot_map pointer of fc_kv_cache points at its start), reference counts
 * [B][S], a free list [B][S] and its tops [B], int32.  0 for B < 1, S < 1 or B S above
 * 2^40. */
size_t fc_slot_state_bytes(int32_t B, int32_t S);

/* Sets up the slot state at kv->slot_map for kv's layout (every row at its own pool row,
 * each frame pool row referenced once, no free row), e.g. with a fresh cache or after
 * fc_cache_update_layers of another layout.  Stream-ordered; `layer` gives the row
 * sizes the validation checks. */
fc_status fc_slot_map_init(fc_ctx *ctx, const fc_layer_desc *layer, const fc_kv_cache *kv,
                           int32_t B, void *stream);

/* fc_cache_step flags */
#define FC_ADVANCE_WINDOW 1  /* kv->head = (kv->head + 1) mod window before anything else */
#define FC_REMAP 2           /* then fc_cache_update on the (advanced) layout */

/* The step's cache preparation for one layer with the window advance done by the library
 * (Sec. 4.1: the frame window moves on, reused tokens take their aligned sources' rows):
 * flags FC_ADVANCE_WINDOW and/or FC_REMAP.  kv->head is written on the host (the descriptor
 * is the caller's); the arguments of FC_REMAP are those of fc_cache_update (shift,
 * reuse_mask, y_prev, y_cur and grid_w are not read without it).  Flags outside the two
 * bits, or none, and a head outside [0, window) are FC_ERR_INVALID_ARG.  On any error
 * kv->head is left as it was: it is written only once the remap has been launched. */
fc_status fc_cache_step(fc_ctx *ctx, const fc_layer_desc *layer, fc_kv_cache *kv,
                        const uint16_t *y_prev, uint16_t *y_cur, const int32_t *shift,
                        const uint8_t *reuse_mask, int32_t grid_w, int32_t flags, int32_t B,
                        void *stream);

/* The partial-recompute decoder layer for B batch items (Sec. 4.1: the tokens that are
 * not reused are recomputed; the per-step computation flow of Sec. 5.2).
 *   x_cur:         [B][N][d_model] bf16 layer input of the current frame's tokens;
 *                  only rows listed in recompute_idx are read;
 *   recompute_idx: [B][N] ascending token ids, n_recompute: [B] (from fc_select);
 *   kv:            this layer's cache; the K/V rows of recomputed tokens in the
 *                  current slot are written, every row is attended;
 *   y_cur:         [B][N][d_model] bf16 output cache; only recomputed rows are written.
 * Queries attend causally by position; QKV of all recomputed tokens is written
 * before any attention, so they see each other's new keys. */
fc_status fc_layer_forward(fc_ctx *ctx, const fc_layer_desc *layer, const fc_kv_cache *kv,
                           const uint16_t *x_cur, const int32_t *recompute_idx,
                           const int32_t *n_recompute, uint16_t *y_cur, int32_t B,
                           void *stream);

/* The vision-encoder side of the partial recompute (Sec. 4.1: a flushed or refreshed
 * token goes through the vision encoder again; a reused one keeps its cached results),
 * for one block.  The patches of the merged tokens recompute_idx[b][0 .. n_recompute[b])
 * (the selection's ids, ascending) go through the block: their raw k, v are written to
 * the cache, their queries attend to every key of their window (cached keys of reused
 * patches, new ones of recomputed patches; keys rotated at their patch position), and
 * their output rows are written to y.  Other rows of y and of the cache are untouched.
 *   x, y: [B][grid_h grid_w merge^2][d_model] bf16 (device), token-major patch rows.
 *   Capacity: the rows, B grid_h grid_w merge^2, use the layer workspace of the context
 *   (each buffer's rows x width within max_batch max_tokens rows x its cap width);
 *   patch grid sides up to 128.  Stream-ordered; allocates nothing. */
fc_status fc_vit_block_forward(fc_ctx *ctx, const fc_vit_desc *layer, const fc_vit_cache *cache,
                               const uint16_t *x, const int32_t *recompute_idx,
                               const int32_t *n_recompute, uint16_t *y, int32_t B, void *stream);

/* The encoder cache's preparation for a new frame (Sec. 4.1 / Eq. 4-2 at patch level):
 * every reused merged token takes the merge^2 patch rows of K, V (from the cache, which
 * holds the previous frame, or from cache->k_prev / v_prev) and of the outputs (y_prev
 * into y_cur) of its source token (I + di, J + dj).  shift [B][2], reuse_mask
 * [B][grid_h grid_w]: from fc_select with the same merge.  y_prev, y_cur:
 * [B][patches][d_model] bf16, non-overlapping, or both NULL (no output rows are moved: a block
 * reads only the recomputed rows of its input, the merger only the recomputed tokens). */
fc_status fc_vit_cache_update(fc_ctx *ctx, const fc_vit_desc *layer, const fc_vit_cache *cache,
                              const uint16_t *y_prev, uint16_t *y_cur, const int32_t *shift,
                              const uint8_t *reuse_mask, int32_t B, void *stream);

/* The patch merger for the recomputed merged tokens only (it acts on each token alone;
 * Sec. 2.1 merged visual tokens, Sec. 4.1 recompute): the language-model input rows
 * x_out[b][recompute_idx[b][j]] for j < n_recompute[b]; other rows are untouched.
 *   y:     [B][n_tokens merge^2][d_model] bf16, the last vision block's outputs
 *          (token-major patch rows);
 *   recompute_idx: [B][n_tokens], n_recompute: [B] (from fc_select with this merge);
 *   x_out: [B][n_tokens][d_out] bf16.
 *   Capacity: 2 B n_tokens hidden <= max_batch max_tokens max_ffn; the split-K
 *   partials within the context's partial-sum workspace (FC_ERR_CAPACITY otherwise).
 * Stream-ordered; allocates nothing. */
fc_status fc_vit_merger_forward(fc_ctx *ctx, const fc_merger_desc *merger, const uint16_t *y,
                                const int32_t *recompute_idx, const int32_t *n_recompute,
                                uint16_t *x_out, int32_t n_tokens, int32_t B, void *stream);

/* Pixel-resolution phase correlation: Eq. 4-1 (Sec. 4.1) with the feature maps taken
 * as the frames' full-resolution BT.601 luma (float64).  The displacement is the first
 * maximum (row-major) of Re F^-1(C), C = X / |X|, X = F(Y_prev) conj(F(Y_cur)), with bins
 * |X| <= 1e-9 max|X| set to 0, wrapped to (-N/2, N/2]; each axis is then refined by the
 * vertex of the parabola through the peak and its two circular neighbours on that axis.
 * Token (I, J) of the current frame shows the content of previous-frame pixel
 * position + (di, dj).
 *   frames_prev, frames_cur: [B][3][H][W] float32 (device); frames_prev may be NULL
 *                (an all-zero previous frame: shift (0, 0)).
 *   H, W:        each 7 * 2^k with 14 <= H, W <= 896 (e.g. 224, 448, 896), within caps;
 *                otherwise FC_ERR_UNSUPPORTED / FC_ERR_CAPACITY.
 *   shift_px:    [B][2] float64 (di, dj) sub-pixel displacement (device, caller-owned).
 *   peak:        [B][2] int32 integer peak (di, dj), or NULL.
 *   response:    [B][H][W] float64 phase-correlation surface, or NULL.
 * The first call on a context allocates its workspace (B H (W/2 + 1) 32 bytes plus row
 * and strip maxima at the caps' sizes); later calls allocate nothing.  Stream-ordered. */
fc_status fc_phase_correlate(fc_ctx *ctx, const float *frames_prev, const float *frames_cur,
                             int32_t B, int32_t H, int32_t W, double *shift_px, int32_t *peak,
                             double *response, void *stream);

/* Pixel-resolution phase correlation after a rotation estimate (Fourier-Mellin): the
 * magnitude spectra of both frames' luma, weighted by (1 - X)(2 - X) with
 * X = cos(pi f_y) cos(pi f_x) (f: signed frequency in cycles per pixel), are sampled
 * bilinearly at H angles i pi / H and min(H, W) / 2 radii R^(j / (min(H, W) / 2)),
 * R = min(H, W) / 2 - 1; Eq. 4-1 on those maps (as fc_phase_correlate, sub-sample peak)
 * gives the angular offset d, and the rotation of the current frame relative to the
 * previous one is a = -d pi / H (radians, in (-pi/2, pi/2]; counter-clockwise in
 * (column, row) coordinates).  The current frame's luma is rotated back about the
 * centre ((H-1)/2, (W-1)/2), bilinear, 0 outside, and Eq. 4-1 on the pair gives
 * shift_px, the displacement of the frame centre.
 *   frames_prev, frames_cur: [B][3][H][W] float32 (device); frames_prev may be NULL.
 *   H, W: 7 * 2^k up to 896 with min(H, W) >= 28, within caps.
 *   angle: [B] float64 or NULL; shift_px: [B][2] float64 (device, caller-owned).
 * Shares the workspace of fc_phase_correlate (allocated at the first call of either). */
fc_status fc_phase_correlate_rotation(fc_ctx *ctx, const float *frames_prev,
                                      const float *frames_cur, int32_t B, int32_t H, int32_t W,
                                      double *angle, double *shift_px, void *stream);

/* Debug mode (process-wide): after every kernel launch the library waits for the
 * launch stream and reports an error raised while the kernel ran as FC_ERR_HIP from
 * the call that launched it, with the kernel's name in fc_last_error().  Streams under
 * graph capture are not waited for.  The mode starts on when the environment variable
 * FC_DEBUG holds anything but "" or "0" as the library loads.  on = 1 / 0 sets it, a
 * negative value leaves it; returns the previous mode.  Outputs are the same either way. */
int32_t fc_debug(int32_t on);

/* Kernel timing with HIP events recorded on the launch stream around every
 * kernel the context launches (off by default). */
fc_status fc_profile_enable(fc_ctx *ctx, int32_t on);
/* Restrict that timing to the launches of kernel `name` (host string, copied);
 * NULL times every kernel again.  Fewer events keep the timed stream closer to
 * an untimed one. */
fc_status fc_profile_only(fc_ctx *ctx, const char *name);
/* Wait for the recorded events and return the summed duration and launch count
 * of kernel `name` (host string) since the last reset; reset=1 clears all records. */
fc_status fc_profile_read(fc_ctx *ctx, const char *name, double *total_ms, int64_t *launches,
                          int32_t reset);

#ifdef __cplusplus
}
#endif
#endif /* FREQCACHE_H */
