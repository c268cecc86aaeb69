// Internal declarations shared by the FreqCache HIP translation units.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <string>
#include <vector>

#include "../../include/freqcache.h"

namespace fc {

// ----------------------------------------------------------------------------- errors
void set_error(const char *fmt, ...);
fc_status fail(fc_status st, const char *fmt, ...);

#define FC_HIP_TRY(expr)                                                                  \
  do {                                                                                    \
    hipError_t _e = (expr);                                                               \
    if (_e != hipSuccess)                                                                 \
      return ::fc::fail(FC_ERR_HIP, "%s failed: %s (%s:%d)", #expr, hipGetErrorString(_e), \
                        __FILE__, __LINE__);                                              \
  } while (0)

// Check after a kernel launch: the launch error and, in debug mode, the stream's
// completion, so that a fault inside the kernel surfaces as FC_ERR_HIP from the call
// that launched it.  Streams under graph capture are not waited for.
hipError_t after_launch(hipStream_t st);
bool debug_mode();

#define FC_LAUNCH_OK(st, what)                                                            \
  do {                                                                                    \
    hipError_t _e = ::fc::after_launch(st);                                               \
    if (_e != hipSuccess)                                                                 \
      return ::fc::fail(FC_ERR_HIP, "%s: %s%s", what, hipGetErrorString(_e),              \
                        ::fc::debug_mode() ? " (debug mode: found when the stream drained)" \
                                           : "");                                         \
  } while (0)

// ----------------------------------------------------------------------------- sizes
constexpr int kPatch = 14;          // the transform kernels are specialised for P = 14
constexpr int kBins = 100;          // unique DFT amplitude bins of a real 14x14 patch
constexpr int kMaxTokens = 1024;    // token-grid / top-K kernels hold one frame in LDS
constexpr int kGemmBK = 64;        // K step of the layer GEMMs (dims must be multiples)
constexpr int kMaxSplits = 16;
// Layer calls with at least this many token slots (B * N) run the large-M path:
// square MFMA tiles with fused epilogues and keys rotated once per call.
constexpr long kBigRows = 2048;
constexpr long kPlainBigRows = 512;  // rows from which run_plain_gemm takes the 256 x 256 tiles

// ----------------------------------------------------------------------------- context
struct ProfRec {
  const char *name;
  hipEvent_t start, stop;
};

}  // namespace fc

struct fc_ctx {
  int device = 0;
  fc_caps caps{};
  int num_cus = 0;
  // selection workspace
  unsigned char *spec = nullptr;   // spectra of two frame batches (prev, cur), FrameSpectra layout
  size_t spec_half = 0;            // bytes of one
  double *penergy = nullptr;   // [B][Np] per-patch high-pass DCT energy (current frame)
  double *pdot = nullptr;      // [B][3][Np] per-patch spectral products (dot, |cur|^2, |src|^2)
  // layer workspace
  uint16_t *qbuf = nullptr;    // [rows][qkv-wide] pre-RoPE queries, bf16
  uint16_t *attn = nullptr;    // [rows][n_heads*hd] attention output, bf16
  float *h1 = nullptr;         // [rows][d] post-attention residual stream
  uint16_t *hb = nullptr;      // [rows][d] bf16 copy of h1 (SwiGLU input)
  float *ssq = nullptr;        // [rows][parts] partial sums of squares of h1 per row
  uint16_t *act = nullptr;     // [rows][ffn] SwiGLU activation, bf16
  float *part = nullptr;       // split-K / split-KV partial sums
  size_t part_elems = 0;
  float2 *rope = nullptr;      // [max_seq][64] (cos, sin)
  int rope_hd = 0, rope_seq = 0;
  double rope_theta = 0.0;
  uint16_t *stage = nullptr;   // [B][N][kv row] staging copy for the W == 1 remap
  size_t stage_elems = 0;
  uint16_t *krot = nullptr;    // [B][S][kv row] rotated keys (many-row layer calls only)
  size_t krot_elems = 0;
  unsigned char *pix = nullptr;  // pixel phase-correlation workspace, allocated at first use
  size_t pix_bytes = 0;
  int32_t *vit_rows = nullptr;  // [max_batch + 1] recomputed patch rows per item (vision
                                // block), then the split count of the last many-row GEMM
  float2 *vit_rope = nullptr;   // [128][32] vision rotary (cos, sin) by position, frequency
  uint16_t *vlog = nullptr;     // [B][S][kv row] values in row order (slot-mapped caches,
  size_t vlog_elems = 0;        // many-row layer calls only), allocated at first use
  // kernel timing
  bool prof = false;
  std::string prof_only;       // empty: time every kernel
  std::vector<fc::ProfRec> recs;
  std::vector<hipEvent_t> pool;
};

namespace fc {

// Event bracket around one launch when profiling is on.
struct ProfScope {
  fc_ctx *ctx;
  hipStream_t st;
  hipEvent_t stop = nullptr;
  ProfScope(fc_ctx *c, hipStream_t s, const char *name);
  ~ProfScope();
};

// ----------------------------------------------------------------------------- launchers
// Spectra of one batch of frames: per-patch DFT amplitudes in 16-patch chunks
// [B][patch row][chunk][kBins][16] and per-patch mean luma [B][Np].  The layout of the
// carried selection state of fc_select_carry.
struct FrameSpectra {
  float *amp;
  double *pmean;
};
// Workspace of the pixel-resolution phase correlation (pixpc.hip): the half-plane
// spectra of both frames [B][H][W/2 + 1] (sa later holds the cross power and its inverse
// column transforms; sb the response surface when the caller gives no buffer), per-row
// maxima and their columns, per-strip largest |X|, and the sub-pixel shifts [B][2].
struct PixWs {
  double2 *sa = nullptr, *sb = nullptr;
  double *rowmax = nullptr;
  int *rowarg = nullptr;
  double *bmax = nullptr;
  double *shift_px = nullptr;
  // rotation only: weighted magnitude spectra, log-polar maps, rotated-back luma
  double *mag = nullptr, *lp = nullptr, *yrot = nullptr;
};
bool pix_size_ok(int n);                       // n = 7 2^k, 14 <= n <= 896
bool pix_rot_size_ok(int H, int W);            // and min(H, W) / 2 too
size_t pix_ws_bytes(long B, long H, long W, bool rot);
PixWs pix_ws_at(void *base, long B, long H, long W, bool rot);
// Eq. 4-1 on full-resolution luma for B pairs (prev may be null: an all-zero frame).
// shift_px [B][2] (null: the workspace's), peak [B][2] integer peak (may be null),
// resp [B][H][W] response surface (may be null), tok_shift [B][2] the displacement in
// whole tokens of tp pixels, (0, 0) with zero_shift (may be null).
fc_status launch_pixel_pc(fc_ctx *ctx, const PixWs &ws, const float *prev, const float *cur,
                          int B, int H, int W, double *shift_px, int32_t *peak, double *resp,
                          int32_t *tok_shift, int tp, bool zero_shift, hipStream_t st);
// The same after finding the current frame's rotation (angle [B], may be null) and undoing
// it; shift_px is then the displacement of the image centre.  ws from pix_ws_at(rot=true).
fc_status launch_pixel_pc_rot(fc_ctx *ctx, const PixWs &ws, const float *prev, const float *cur,
                              int B, int H, int W, double *angle, double *shift_px,
                              int32_t *tok_shift, int tp, bool zero_shift, hipStream_t st);

// Selection workspace: spectra of the previous and the current frames, per-patch
// high-pass energies (current frame) and spectral products; pix only with align_pixel.
struct SelectWs {
  FrameSpectra prev, cur;
  double *penergy;   // [B][Np]
  double *pdot;      // [B][3][Np]
  PixWs pix;
};
// Bytes of one frame batch's spectra (256-B aligned parts) and of the whole workspace.
struct SpectraBytes {
  size_t amp, pmean, total;
};
SpectraBytes spectra_bytes(long B, long H, long W);
FrameSpectra spectra_at(void *base, long B, long H, long W);
struct SelectWsBytes {
  size_t spectra, penergy, pdot, total;   // spectra: one frame batch (two are used)
};
SelectWsBytes select_ws_bytes(long B, long H, long W);

// Argument checks shared by the selection entry points (synchronous, no device work).
fc_status check_select_args(const fc_select_params *prm, const float *cur,
                            const fc_select_out *out, int B, int H, int W, const char *who);

// ctx may be null (no kernel timing).  carried: the previous frame's spectra are
// already in ws.prev (prev pixels unused); otherwise both frames are transformed.
fc_status launch_select(fc_ctx *ctx, const SelectWs &ws, const fc_select_params &prm,
                        const float *prev, const float *cur, int B, int H, int W,
                        const fc_select_out &out, hipStream_t st, bool carried = false);
// The same on the calling thread's current device, with the workspace in the library's
// static device scratch array (no allocation).
fc_status launch_select_noalloc(const fc_select_params &prm, const float *prev,
                                const float *cur, int B, int H, int W,
                                const fc_select_out &out, hipStream_t st);
size_t noalloc_scratch_bytes();

// Slot-map state of B items with S cache rows (slotmap.hip): map [B][S], ref [B][S],
// free [B][S], top [B], int32, in that order.
struct SlotState {
  int32_t *map, *ref, *free, *top;
};
__host__ __device__ inline SlotState slot_state_at(int32_t *base, long B, long S) {
  return SlotState{base, base + B * S, base + 2 * B * S, base + 3 * B * S};
}
size_t slot_state_bytes(long B, long S);
fc_status launch_slot_init(fc_ctx *ctx, const fc_kv_cache &kv, int B, hipStream_t st);
// The step's map update for all layers sharing kv.slot_map (window already advanced).
fc_status launch_slot_remap(fc_ctx *ctx, const fc_kv_cache &kv, const int32_t *shift,
                            const uint8_t *reuse, int grid_w, int B, hipStream_t st);
// Pool row of cache row r of item b: the map's entry (clamped into the item's rows), or
// r itself without a map.
__device__ __forceinline__ int pool_row(const int32_t *map, int b, int S, int r) {
  if (!map) return r;
  const int p = map[(long)b * S + r];
  return p < 0 ? 0 : (p >= S ? S - 1 : p);
}

// Split-K partial sums of A[B N][K] W[Nout][K]^T over the first nrec[b] rows of each
// item, no epilogue; K a multiple of 64, Nout of 16.  Few rows: the weight-streaming GEMM,
// part = C[split][B N][Nout], *splits = its split count, *dsplits_used = null, *tiles = 0.
// Many rows (and dsplits given): the 256 x 256-tile GEMM over the rows packed across
// items (item b's rows after those of items < b), part = [split][V][ceil(Nout / 256)]
// tiles of [256 packed rows][256 columns], V = ceil(packed rows / 256); its split count
// (at most 8) is decided on the device and written to *dsplits; *splits = 8,
// *dsplits_used = dsplits and *tiles = 1.
fc_status run_plain_gemm(fc_ctx *ctx, hipStream_t st, const char *name, const uint16_t *A,
                         const uint16_t *W, int K, int Nout, int N, const int32_t *nrec,
                         float *part, int B, int *splits, int *dsplits,
                         const int **dsplits_used, int *tiles);

// Vision-encoder block with partial recompute and its cache update (vit.hip).
// Reused tokens' K/V rows (and output rows, when y_prev is given) copied from a previous
// frame's cache [B][N][kvw] into a distinct current one, token (I, J) from (I + di, J + dj)
// (the layer remap with source and destination in separate buffers: no staging).
fc_status launch_remap_copy(fc_ctx *ctx, const uint16_t *ksrc, const uint16_t *vsrc, uint16_t *kdst,
                            uint16_t *vdst, const uint16_t *y_prev, uint16_t *y_cur, int N, int kvw,
                            int d, int grid_w, const int32_t *shift, const uint8_t *reuse, int B,
                            hipStream_t st);
fc_status launch_vit_block(fc_ctx *ctx, const fc_vit_desc &L, const fc_vit_cache &c,
                           const uint16_t *x, const int32_t *idx, const int32_t *nrec,
                           uint16_t *y, int B, hipStream_t st);
fc_status launch_vit_cache_update(fc_ctx *ctx, const fc_vit_desc &L, const fc_vit_cache &c,
                                  const uint16_t *y_prev, uint16_t *y_cur, const int32_t *shift,
                                  const uint8_t *reuse, int B, hipStream_t st);
fc_status launch_vit_merger(fc_ctx *ctx, const fc_merger_desc &M, const uint16_t *y,
                            const int32_t *idx, const int32_t *nrec, uint16_t *x_out, int N,
                            int B, hipStream_t st);

// trail: recompute the text rows after the frames instead of the selected frame tokens
fc_status launch_layer(fc_ctx *ctx, const fc_layer_desc &L, const fc_kv_cache &kv,
                       const uint16_t *x_cur, const int32_t *idx, const int32_t *nrec,
                       uint16_t *y_cur, int B, hipStream_t st, bool trail = false);

fc_status launch_cache_update(fc_ctx *ctx, const fc_layer_desc &L, const fc_kv_cache &kv,
                              const uint16_t *y_prev, uint16_t *y_cur, const int32_t *shift,
                              const uint8_t *reuse, int grid_w, int B, hipStream_t st);
fc_status launch_cache_update_layers(fc_ctx *ctx, const fc_layer_desc &L, int n_layers,
                                     const fc_kv_cache *kvs, const uint16_t *const *y_prev,
                                     uint16_t *const *y_cur, const int32_t *shift,
                                     const uint8_t *reuse, int grid_w, int B, hipStream_t st);

fc_status upload_select_tables();

}  // namespace fc
