// C ABI of the FreqCache hot path: argument validation, context and workspace,
// error reporting and event-based kernel timing.  The kernels live in select.hip
// and layer.hip.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <new>

#include "fc_internal.h"

namespace fc {

static thread_local char g_err[1024] = "";

void set_error(const char *fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
}

fc_status fail(fc_status st, const char *fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof(g_err), fmt, ap);
  va_end(ap);
  return st;
}

// Whether the byte ranges [a, a + n) and [b, b + n) share a byte (both given): a remap
// that reads one while writing the other would race.
static bool overlap(const void *a, const void *b, size_t n) {
  const uintptr_t x = reinterpret_cast<uintptr_t>(a), y = reinterpret_cast<uintptr_t>(b);
  return a && b && x < y + n && y < x + n;
}

// Debug mode: FC_DEBUG set to anything but "" or "0" when the library loads, or fc_debug.
static std::atomic<int> g_debug{[] {
  const char *e = std::getenv("FC_DEBUG");
  return (e && *e && std::strcmp(e, "0") != 0) ? 1 : 0;
}()};

bool debug_mode() { return g_debug.load(std::memory_order_relaxed) != 0; }

hipError_t after_launch(hipStream_t st) {
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || !debug_mode()) return e;
  hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
  if (hipStreamIsCapturing(st, &cs) == hipSuccess && cs != hipStreamCaptureStatusNone)
    return hipSuccess;
  e = hipStreamSynchronize(st);
  return e != hipSuccess ? e : hipGetLastError();
}

ProfScope::ProfScope(fc_ctx *c, hipStream_t s, const char *name) : ctx(c), st(s) {
  if (!ctx || !ctx->prof || (!ctx->prof_only.empty() && ctx->prof_only != name)) return;
  hipEvent_t a, b;
  if (ctx->pool.size() >= 2) {
    a = ctx->pool.back();
    ctx->pool.pop_back();
    b = ctx->pool.back();
    ctx->pool.pop_back();
  } else {
    if (hipEventCreate(&a) != hipSuccess) return;
    if (hipEventCreate(&b) != hipSuccess) {
      hipEventDestroy(a);
      return;
    }
  }
  hipEventRecord(a, st);
  ctx->recs.push_back(ProfRec{name, a, b});
  stop = b;
}

ProfScope::~ProfScope() {
  if (stop) hipEventRecord(stop, st);
}

SpectraBytes spectra_bytes(long B, long H, long W) {
  auto al = [](size_t x) { return (x + 255) & ~(size_t)255; };
  const size_t np = (size_t)(H / kPatch) * (W / kPatch);
  // amplitudes in 16-patch chunks of a patch row (the last chunk of a row padded)
  const size_t np16 = (size_t)(H / kPatch) * ((W / kPatch + 15) / 16) * 16;
  SpectraBytes b;
  b.amp = al((size_t)B * kBins * np16 * sizeof(float));
  b.pmean = al((size_t)B * np * sizeof(double));
  b.total = b.amp + b.pmean;
  return b;
}

FrameSpectra spectra_at(void *base, long B, long H, long W) {
  const SpectraBytes b = spectra_bytes(B, H, W);
  unsigned char *p = static_cast<unsigned char *>(base);
  return FrameSpectra{reinterpret_cast<float *>(p), reinterpret_cast<double *>(p + b.amp)};
}

SelectWsBytes select_ws_bytes(long B, long H, long W) {
  auto al = [](size_t x) { return (x + 255) & ~(size_t)255; };
  const size_t np = (size_t)(H / kPatch) * (W / kPatch);
  SelectWsBytes b;
  b.spectra = spectra_bytes(B, H, W).total;
  b.penergy = al((size_t)B * np * sizeof(double));
  b.pdot = al((size_t)B * 3 * np * sizeof(double));
  b.total = 2 * b.spectra + b.penergy + b.pdot;
  return b;
}

fc_status check_select_args(const fc_select_params *prm, const float *cur,
                            const fc_select_out *out, int B, int H, int W, const char *who) {
  if (!prm || !cur || !out)
    return fail(FC_ERR_INVALID_ARG, "%s: null params, current frames or outputs", who);
  if (!out->sim || !out->energy || !out->reuse_mask || !out->recompute_idx || !out->n_recompute ||
      !out->shift || !out->scalars || !out->counts)
    return fail(FC_ERR_INVALID_ARG, "%s: an output buffer is null", who);
  const fc_select_params &p = *prm;
  if (p.patch != kPatch)
    return fail(FC_ERR_UNSUPPORTED, "%s: patch %d (the library implements P = 14)", who, p.patch);
  if (p.merge < 1 || p.merge > 4) return fail(FC_ERR_INVALID_ARG, "%s: merge %d", who, p.merge);
  if (!(p.alpha_min >= 0 && p.alpha_max <= 1 && p.alpha_min <= p.alpha_max) ||
      !(p.alpha_fixed >= 0 && p.alpha_fixed <= 1) || !(p.lambda_ >= 0) || !std::isfinite(p.tau_mig) ||
      !std::isfinite(p.tau_sim) || (p.no_align != 0 && p.no_align != 1) ||
      (p.no_refresh != 0 && p.no_refresh != 1) || (p.align_pixel != 0 && p.align_pixel != 1) ||
      (p.align_rotation != 0 && p.align_rotation != 1) || (p.align_rotation && !p.align_pixel))
    return fail(FC_ERR_INVALID_ARG, "%s: hyper-parameter out of range", who);
  if (B < 1 || H < 1 || W < 1) return fail(FC_ERR_SHAPE, "%s: B=%d H=%d W=%d", who, B, H, W);
  const int tp = p.patch * p.merge;
  if (H % tp || W % tp)
    return fail(FC_ERR_SHAPE, "%s: H=%d, W=%d not multiples of patch*merge=%d", who, H, W, tp);
  const long M = (long)(H / tp) * (W / tp);
  if (M > kMaxTokens)
    return fail(FC_ERR_UNSUPPORTED, "%s: %ld tokens per frame > %d", who, M, kMaxTokens);
  if (p.align_rotation && !pix_rot_size_ok(H, W))
    return fail(FC_ERR_UNSUPPORTED, "%s: align_rotation needs H and W of the form 7 * 2^k up to "
                "896 with min(H, W) >= 28 (got %dx%d)", who, H, W);
  if (p.align_pixel && (!pix_size_ok(H) || !pix_size_ok(W)))
    return fail(FC_ERR_UNSUPPORTED, "%s: align_pixel needs H and W of the form 7 * 2^k up to 896 "
                "(got %dx%d)", who, H, W);
  return FC_OK;
}

}  // namespace fc

using fc::fail;

namespace {

const char *kVersion = "freqcache-mi355x 0.1 (gfx950)";

template <typename T>
fc_status dev_alloc(T **p, size_t count, const char *what) {
  *p = nullptr;
  if (count == 0) count = 1;
  hipError_t e = hipMalloc(reinterpret_cast<void **>(p), count * sizeof(T));
  if (e != hipSuccess)
    return fail(FC_ERR_HIP, "hipMalloc(%s, %zu bytes): %s", what, count * sizeof(T),
                hipGetErrorString(e));
  return FC_OK;
}

void free_ws(fc_ctx *c) {
  void *ptrs[] = {c->spec, c->penergy, c->pdot, c->qbuf, c->attn,
                  c->h1,  c->hb,    c->act,     c->part,    c->rope, c->stage, c->ssq,
                  c->krot, c->pix, c->vlog, c->vit_rows, c->vit_rope};
  for (void *p : ptrs)
    if (p) hipFree(p);
  for (auto &r : c->recs) {
    hipEventDestroy(r.start);
    hipEventDestroy(r.stop);
  }
  for (auto e : c->pool) hipEventDestroy(e);
  c->recs.clear();
  c->pool.clear();
}

fc_status use_device(fc_ctx *ctx) {
  hipError_t e = hipSetDevice(ctx->device);
  if (e != hipSuccess) return fail(FC_ERR_HIP, "hipSetDevice(%d): %s", ctx->device, hipGetErrorString(e));
  return FC_OK;
}

// The pixel phase-correlation workspace, sized for the context's caps at its first use.
fc_status ensure_pix(fc_ctx *ctx) {
  if (ctx->pix) return FC_OK;
  // sized for the rotation mode, whose parts come after the plain mode's
  const size_t bytes = fc::pix_ws_bytes(ctx->caps.max_batch, ctx->caps.max_height,
                                        ctx->caps.max_width, true);
  hipError_t e = hipMalloc(reinterpret_cast<void **>(&ctx->pix), bytes);
  if (e != hipSuccess) {
    ctx->pix = nullptr;
    return fail(FC_ERR_HIP, "hipMalloc(pixel phase correlation, %zu bytes): %s", bytes,
                hipGetErrorString(e));
  }
  ctx->pix_bytes = bytes;
  return FC_OK;
}

}  // namespace

extern "C" {

const char *fc_version(void) { return kVersion; }

const char *fc_last_error(void) { return fc::g_err; }

fc_status fc_create(fc_ctx **out, int32_t device, const fc_caps *caps) {
  if (!out || !caps) return fail(FC_ERR_INVALID_ARG, "fc_create: null out or caps");
  *out = nullptr;
  const fc_caps &c = *caps;
  if (c.max_batch < 1 || c.max_height < 1 || c.max_width < 1 || c.max_tokens < 1 ||
      c.max_seq < 1 || c.max_d_model < 1 || c.max_ffn < 1 || c.max_qkv < 1)
    return fail(FC_ERR_INVALID_ARG, "fc_create: every cap must be >= 1");
  if (c.max_tokens > fc::kMaxTokens)
    return fail(FC_ERR_UNSUPPORTED, "fc_create: max_tokens %d > %d", c.max_tokens, fc::kMaxTokens);
  int n = 0;
  hipError_t e = hipGetDeviceCount(&n);
  if (e != hipSuccess || n < 1)
    return fail(FC_ERR_NO_DEVICE, "fc_create: no HIP device (%s)",
                e != hipSuccess ? hipGetErrorString(e) : "count 0");
  if (device < 0 || device >= n)
    return fail(FC_ERR_INVALID_ARG, "fc_create: device %d of %d", device, n);
  e = hipSetDevice(device);
  if (e != hipSuccess) return fail(FC_ERR_HIP, "hipSetDevice: %s", hipGetErrorString(e));
  hipDeviceProp_t prop;
  e = hipGetDeviceProperties(&prop, device);
  if (e != hipSuccess) return fail(FC_ERR_HIP, "hipGetDeviceProperties: %s", hipGetErrorString(e));
  if (std::strncmp(prop.gcnArchName, "gfx950", 6) != 0)
    return fail(FC_ERR_UNSUPPORTED, "fc_create: device is %s, the library targets gfx950",
                prop.gcnArchName);

  fc_ctx *ctx = new (std::nothrow) fc_ctx();
  if (!ctx) return fail(FC_ERR_INVALID_ARG, "fc_create: out of host memory");
  ctx->device = device;
  ctx->caps = c;
  ctx->num_cus = prop.multiProcessorCount;
  const size_t B = c.max_batch;
  const size_t rows = B * c.max_tokens;
  const size_t wide = std::max(c.max_qkv, c.max_d_model) + 64;
  const size_t base = rows * wide;
  const size_t cap = (size_t)96 << 20;
  ctx->part_elems = base * std::min<size_t>(fc::kMaxSplits, std::max<size_t>(1, cap / base));
  ctx->stage_elems = B * c.max_tokens * (size_t)c.max_qkv;
  // a kv row is at most a third of a qkv row (n_heads >= n_kv_heads)
  if ((long)rows >= fc::kBigRows) ctx->krot_elems = B * (size_t)c.max_seq * ((c.max_qkv + 2) / 3);
  fc_status st = FC_OK;
  const fc::SelectWsBytes sb = fc::select_ws_bytes(B, c.max_height, c.max_width);
  ctx->spec_half = sb.spectra;
  if ((st = dev_alloc(&ctx->spec, 2 * sb.spectra, "spectra")) != FC_OK ||
      (st = dev_alloc(&ctx->penergy, sb.penergy / sizeof(double), "penergy")) != FC_OK ||
      (st = dev_alloc(&ctx->pdot, sb.pdot / sizeof(double), "pdot")) != FC_OK ||
      (st = dev_alloc(&ctx->qbuf, rows * c.max_qkv, "q")) != FC_OK ||
      (st = dev_alloc(&ctx->attn, rows * c.max_qkv, "attn")) != FC_OK ||
      (st = dev_alloc(&ctx->h1, rows * c.max_d_model, "h1")) != FC_OK ||
      (st = dev_alloc(&ctx->hb, rows * c.max_d_model, "hb")) != FC_OK ||
      (st = dev_alloc(&ctx->ssq, rows * std::max<size_t>(8, (c.max_d_model + 127) / 128), "ssq")) != FC_OK ||
      (st = dev_alloc(&ctx->act, rows * c.max_ffn, "act")) != FC_OK ||
      (st = dev_alloc(&ctx->part, ctx->part_elems, "partials")) != FC_OK ||
      (st = dev_alloc(&ctx->rope, (size_t)c.max_seq * 64, "rope")) != FC_OK ||
      (st = dev_alloc(&ctx->stage, ctx->stage_elems, "stage")) != FC_OK ||
      (ctx->krot_elems && (st = dev_alloc(&ctx->krot, ctx->krot_elems, "rotated keys")) != FC_OK) ||
      (st = dev_alloc(&ctx->vit_rows, B + 1, "vision rows")) != FC_OK ||
      (st = dev_alloc(&ctx->vit_rope, (size_t)128 * 32, "vision rotary table")) != FC_OK ||
      (st = fc::upload_select_tables()) != FC_OK) {
    free_ws(ctx);
    delete ctx;
    return st;
  }
  *out = ctx;
  return FC_OK;
}

fc_status fc_destroy(fc_ctx *ctx) {
  if (!ctx) return fail(FC_ERR_INVALID_ARG, "fc_destroy: null context");
  hipSetDevice(ctx->device);
  hipDeviceSynchronize();
  free_ws(ctx);
  delete ctx;
  return FC_OK;
}

fc_status fc_select(fc_ctx *ctx, const fc_select_params *prm, const float *frames_prev,
                    const float *frames_cur, int32_t B, int32_t H, int32_t W,
                    const fc_select_out *out, void *stream) {
  if (!ctx) return fail(FC_ERR_INVALID_ARG, "fc_select: null context");
  fc_status st = fc::check_select_args(prm, frames_cur, out, B, H, W, "fc_select");
  if (st != FC_OK) return st;
  const int tp = prm->patch * prm->merge;
  const int M = (H / tp) * (W / tp);
  if (B > ctx->caps.max_batch || H > ctx->caps.max_height || W > ctx->caps.max_width ||
      M > ctx->caps.max_tokens)
    return fail(FC_ERR_CAPACITY, "fc_select: B=%d H=%d W=%d N=%d exceed the context caps", B, H, W, M);
  st = use_device(ctx);
  if (st != FC_OK) return st;
  fc::SelectWs ws{fc::spectra_at(ctx->spec, B, H, W),
                  fc::spectra_at(ctx->spec + ctx->spec_half, B, H, W), ctx->penergy, ctx->pdot,
                  {}};
  if (prm->align_pixel) {
    if ((st = ensure_pix(ctx)) != FC_OK) return st;
    ws.pix = fc::pix_ws_at(ctx->pix, B, H, W, prm->align_rotation != 0);
  }
  return fc::launch_select(ctx, ws, *prm, frames_prev, frames_cur, B, H, W, *out,
                           reinterpret_cast<hipStream_t>(stream));
}

size_t fc_select_state_bytes(int32_t B, int32_t H, int32_t W) {
  if (B < 1 || H < fc::kPatch || W < fc::kPatch) return 0;
  return fc::spectra_bytes(B, H, W).total;
}

fc_status fc_select_carry(fc_ctx *ctx, const fc_select_params *prm, const void *state_prev,
                          const float *frames_cur, void *state_cur, int32_t B, int32_t H,
                          int32_t W, const fc_select_out *out, void *stream) {
  if (!ctx) return fail(FC_ERR_INVALID_ARG, "fc_select_carry: null context");
  fc_status st = fc::check_select_args(prm, frames_cur, out, B, H, W, "fc_select_carry");
  if (st != FC_OK) return st;
  if (!state_cur) return fail(FC_ERR_INVALID_ARG, "fc_select_carry: null state_cur");
  if (prm->align_pixel)
    return fail(FC_ERR_UNSUPPORTED, "fc_select_carry: align_pixel needs the previous frame's "
                "pixels; use fc_select");
  if (state_cur == state_prev || fc::overlap(state_prev, state_cur, fc_select_state_bytes(B, H, W)))
    return fail(FC_ERR_INVALID_ARG, "fc_select_carry: state_prev and state_cur overlap");
  const int tp = prm->patch * prm->merge;
  const int M = (H / tp) * (W / tp);
  if (B > ctx->caps.max_batch || H > ctx->caps.max_height || W > ctx->caps.max_width ||
      M > ctx->caps.max_tokens)
    return fail(FC_ERR_CAPACITY, "fc_select_carry: B=%d H=%d W=%d N=%d exceed the context caps",
                B, H, W, M);
  st = use_device(ctx);
  if (st != FC_OK) return st;
  // without a previous state the previous frame is an all-zero frame, transformed into
  // the context's own previous half
  const bool carried = state_prev != nullptr;
  const fc::SelectWs ws{carried ? fc::spectra_at(const_cast<void *>(state_prev), B, H, W)
                                : fc::spectra_at(ctx->spec, B, H, W),
                        fc::spectra_at(state_cur, B, H, W), ctx->penergy, ctx->pdot, {}};
  return fc::launch_select(ctx, ws, *prm, nullptr, frames_cur, B, H, W, *out,
                           reinterpret_cast<hipStream_t>(stream), carried);
}

fc_status fc_select_noalloc(const fc_select_params *prm, const float *frames_prev,
                            const float *frames_cur, int32_t B, int32_t H, int32_t W,
                            const fc_select_out *out, void *stream) {
  fc_status st = fc::check_select_args(prm, frames_cur, out, B, H, W, "fc_select_noalloc");
  if (st != FC_OK) return st;
  const size_t need = fc::select_ws_bytes(B, H, W).total;
  if (need > fc::noalloc_scratch_bytes())
    return fail(FC_ERR_CAPACITY,
                "fc_select_noalloc: B=%d pairs of %dx%d frames need %zu bytes of scratch, "
                "the static scratch holds %zu",
                B, H, W, need, fc::noalloc_scratch_bytes());
  return fc::launch_select_noalloc(*prm, frames_prev, frames_cur, B, H, W, *out,
                                   reinterpret_cast<hipStream_t>(stream));
}

fc_status fc_phase_correlate(fc_ctx *ctx, const float *frames_prev, const float *frames_cur,
                             int32_t B, int32_t H, int32_t W, double *shift_px, int32_t *peak,
                             double *response, void *stream) {
  if (!ctx) return fail(FC_ERR_INVALID_ARG, "fc_phase_correlate: null context");
  if (!frames_cur || !shift_px)
    return fail(FC_ERR_INVALID_ARG, "fc_phase_correlate: null current frames or shift output");
  if (B < 1 || H < 1 || W < 1) return fail(FC_ERR_SHAPE, "fc_phase_correlate: B=%d H=%d W=%d", B, H, W);
  if (!fc::pix_size_ok(H) || !fc::pix_size_ok(W))
    return fail(FC_ERR_UNSUPPORTED, "fc_phase_correlate: H and W must be 7 * 2^k up to 896 "
                "(got %dx%d)", H, W);
  if (B > ctx->caps.max_batch || H > ctx->caps.max_height || W > ctx->caps.max_width)
    return fail(FC_ERR_CAPACITY, "fc_phase_correlate: B=%d H=%d W=%d exceed the context caps", B, H, W);
  fc_status st = use_device(ctx);
  if (st != FC_OK) return st;
  if ((st = ensure_pix(ctx)) != FC_OK) return st;
  return fc::launch_pixel_pc(ctx, fc::pix_ws_at(ctx->pix, B, H, W, false), frames_prev, frames_cur, B, H,
                             W, shift_px, peak, response, nullptr, 1, false,
                             reinterpret_cast<hipStream_t>(stream));
}

fc_status fc_phase_correlate_rotation(fc_ctx *ctx, const float *frames_prev,
                                      const float *frames_cur, int32_t B, int32_t H, int32_t W,
                                      double *angle, double *shift_px, void *stream) {
  if (!ctx) return fail(FC_ERR_INVALID_ARG, "fc_phase_correlate_rotation: null context");
  if (!frames_cur || !shift_px)
    return fail(FC_ERR_INVALID_ARG, "fc_phase_correlate_rotation: null current frames or shift output");
  if (B < 1 || H < 1 || W < 1)
    return fail(FC_ERR_SHAPE, "fc_phase_correlate_rotation: B=%d H=%d W=%d", B, H, W);
  if (!fc::pix_rot_size_ok(H, W))
    return fail(FC_ERR_UNSUPPORTED, "fc_phase_correlate_rotation: H and W must be 7 * 2^k up to 896 "
                "with min(H, W) >= 28 (got %dx%d)", H, W);
  if (B > ctx->caps.max_batch || H > ctx->caps.max_height || W > ctx->caps.max_width)
    return fail(FC_ERR_CAPACITY, "fc_phase_correlate_rotation: B=%d H=%d W=%d exceed the context caps",
                B, H, W);
  fc_status st = use_device(ctx);
  if (st != FC_OK) return st;
  if ((st = ensure_pix(ctx)) != FC_OK) return st;
  return fc::launch_pixel_pc_rot(ctx, fc::pix_ws_at(ctx->pix, B, H, W, true), frames_prev,
                                 frames_cur, B, H, W, angle, shift_px, nullptr, 1, false,
                                 reinterpret_cast<hipStream_t>(stream));
}

static fc_status check_layer(fc_ctx *ctx, const fc_layer_desc *L, const fc_kv_cache *kv, int B,
                             const char *who) {
  if (!L || !kv) return fail(FC_ERR_INVALID_ARG, "%s: null layer or cache descriptor", who);
  if (L->d_model < 1 || L->n_heads < 1 || L->n_kv_heads < 1 || L->head_dim < 1 || L->d_ffn < 1)
    return fail(FC_ERR_INVALID_ARG, "%s: non-positive layer dimension", who);
  if (L->n_heads % L->n_kv_heads)
    return fail(FC_ERR_SHAPE, "%s: n_kv_heads %d does not divide n_heads %d", who, L->n_kv_heads,
                L->n_heads);
  if (L->d_model > 8192)
    return fail(FC_ERR_UNSUPPORTED, "%s: d_model %d > 8192", who, L->d_model);
  if (L->n_heads > 128)
    return fail(FC_ERR_UNSUPPORTED, "%s: n_heads %d > 128", who, L->n_heads);
  if (L->head_dim > 256)
    return fail(FC_ERR_UNSUPPORTED, "%s: head_dim %d > 256", who, L->head_dim);
  if (L->d_model % fc::kGemmBK || L->d_ffn % fc::kGemmBK || ((long)L->n_heads * L->head_dim) % fc::kGemmBK)
    return fail(FC_ERR_SHAPE, "%s: d_model, d_ffn and n_heads*head_dim must be multiples of %d", who,
                fc::kGemmBK);
  if (!(L->rms_eps > 0) || !(L->rope_theta > 1))
    return fail(FC_ERR_INVALID_ARG, "%s: rms_eps must be > 0 and rope_theta > 1", who);
  if (!kv->k || !kv->v) return fail(FC_ERR_INVALID_ARG, "%s: null K or V cache", who);
  if (kv->text_tokens < 0 || kv->frame_tokens < 1 || kv->window < 1 || kv->head < 0 ||
      kv->head >= kv->window)
    return fail(FC_ERR_INVALID_ARG, "%s: bad cache layout T=%d N=%d W=%d head=%d", who,
                kv->text_tokens, kv->frame_tokens, kv->window, kv->head);
  if (kv->trail_tokens < 0)
    return fail(FC_ERR_INVALID_ARG, "%s: trail_tokens %d", who, kv->trail_tokens);
  const long S = (long)kv->text_tokens + (long)kv->window * kv->frame_tokens + kv->trail_tokens;
  const long qkv = ((long)L->n_heads + 2L * L->n_kv_heads) * L->head_dim;
  const int *ms = kv->mrope_section;
  if (ms[0] || ms[1] || ms[2]) {
    if (ms[0] < 0 || ms[1] < 0 || ms[2] < 0 || ms[0] % 8 || ms[1] % 8 || ms[2] % 8 ||
        (long)ms[0] + ms[1] + ms[2] != L->head_dim / 2)
      return fail(FC_ERR_INVALID_ARG, "%s: M-RoPE sections %d/%d/%d must be multiples of 8 "
                  "summing to head_dim/2 = %d", who, ms[0], ms[1], ms[2], L->head_dim / 2);
    if (kv->grid_w < 1 || kv->frame_tokens % kv->grid_w)
      return fail(FC_ERR_SHAPE, "%s: grid_w %d does not divide N=%d", who, kv->grid_w,
                  kv->frame_tokens);
  }
  const fc_caps &c = ctx->caps;
  if (B < 1) return fail(FC_ERR_SHAPE, "%s: B=%d", who, B);
  if (B > c.max_batch || kv->frame_tokens > c.max_tokens || kv->trail_tokens > c.max_tokens ||
      S > c.max_seq || L->d_model > c.max_d_model ||
      L->d_ffn > c.max_ffn || qkv > c.max_qkv)
    return fail(FC_ERR_CAPACITY, "%s: B=%d N=%d S=%ld d=%d ffn=%d qkv=%ld exceed the context caps",
                who, B, kv->frame_tokens, S, L->d_model, L->d_ffn, qkv);
  // the GEMMs address weights and activation rows with 32-bit element offsets
  const long wmax = std::max({(long)qkv, (long)L->d_model, (long)L->d_ffn}) *
                    std::max({(long)L->d_model, (long)L->d_ffn, (long)L->n_heads * L->head_dim});
  if (wmax >= (1L << 32))
    return fail(FC_ERR_UNSUPPORTED, "%s: weight matrices of 2^32 or more elements", who);
  if (kv->slot_map && S * (long)L->n_kv_heads * L->head_dim * 2 >= (1L << 32))
    return fail(FC_ERR_UNSUPPORTED, "%s: a slot-mapped item's K or V rows must span less than 4 GiB", who);
  const long widest = std::max({(long)L->d_model, (long)L->d_ffn, (long)L->n_heads * L->head_dim});
  if ((long)B * kv->frame_tokens * widest >= (1L << 32))
    return fail(FC_ERR_CAPACITY, "%s: B*N*%ld activation elements exceed 2^32", who, widest);
  return FC_OK;
}

fc_status fc_layer_forward(fc_ctx *ctx, const fc_layer_desc *layer, const fc_kv_cache *kv,
                           const uint16_t *x_cur, const int32_t *recompute_idx,
                           const int32_t *n_recompute, uint16_t *y_cur, int32_t B,
                           void *stream) {
  if (!ctx) return fail(FC_ERR_INVALID_ARG, "fc_layer_forward: null context");
  fc_status st = check_layer(ctx, layer, kv, B, "fc_layer_forward");
  if (st != FC_OK) return st;
  const fc_layer_desc &L = *layer;
  if (!x_cur || !recompute_idx || !n_recompute || !y_cur)
    return fail(FC_ERR_INVALID_ARG, "fc_layer_forward: null activation or index buffer");
  if (!L.w_qkv || !L.b_qkv || !L.w_o || !L.w_gate || !L.w_up || !L.w_down || !L.g_attn || !L.g_mlp)
    return fail(FC_ERR_INVALID_ARG, "fc_layer_forward: null weight pointer");
  if (!((L.head_dim == 128 && (L.n_heads / L.n_kv_heads == 7 || L.n_heads / L.n_kv_heads == 1 ||
                               L.n_heads / L.n_kv_heads == 4)) ||
        (L.head_dim == 64 && (L.n_heads / L.n_kv_heads == 1 || L.n_heads / L.n_kv_heads == 2))))
    return fail(FC_ERR_UNSUPPORTED, "fc_layer_forward: head_dim %d with %d query heads per kv head",
                L.head_dim, L.n_heads / L.n_kv_heads);
  if ((long)kv->text_tokens + (long)kv->window * kv->frame_tokens + kv->trail_tokens >
      (long)ctx->caps.max_seq)
    return fail(FC_ERR_CAPACITY, "fc_layer_forward: sequence exceeds max_seq");
  st = use_device(ctx);
  if (st != FC_OK) return st;
  return fc::launch_layer(ctx, L, *kv, x_cur, recompute_idx, n_recompute, y_cur, B,
                          reinterpret_cast<hipStream_t>(stream));
}

fc_status fc_layer_forward_trail(fc_ctx *ctx, const fc_layer_desc *layer, const fc_kv_cache *kv,
                                 const uint16_t *x_trail, uint16_t *y_trail, int32_t B,
                                 void *stream) {
  if (!ctx) return fail(FC_ERR_INVALID_ARG, "fc_layer_forward_trail: null context");
  fc_status st = check_layer(ctx, layer, kv, B, "fc_layer_forward_trail");
  if (st != FC_OK) return st;
  const fc_layer_desc &L = *layer;
  if (kv->trail_tokens < 1)
    return fail(FC_ERR_INVALID_ARG, "fc_layer_forward_trail: the cache has no trailing text");
  if (!x_trail || !y_trail)
    return fail(FC_ERR_INVALID_ARG, "fc_layer_forward_trail: null activation buffer");
  if (!L.w_qkv || !L.b_qkv || !L.w_o || !L.w_gate || !L.w_up || !L.w_down || !L.g_attn || !L.g_mlp)
    return fail(FC_ERR_INVALID_ARG, "fc_layer_forward_trail: null weight pointer");
  if (!((L.head_dim == 128 && (L.n_heads / L.n_kv_heads == 7 || L.n_heads / L.n_kv_heads == 1 ||
                               L.n_heads / L.n_kv_heads == 4)) ||
        (L.head_dim == 64 && (L.n_heads / L.n_kv_heads == 1 || L.n_heads / L.n_kv_heads == 2))))
    return fail(FC_ERR_UNSUPPORTED, "fc_layer_forward_trail: head_dim %d with %d query heads per kv head",
                L.head_dim, L.n_heads / L.n_kv_heads);
  st = use_device(ctx);
  if (st != FC_OK) return st;
  return fc::launch_layer(ctx, L, *kv, x_trail, nullptr, nullptr, y_trail, B,
                          reinterpret_cast<hipStream_t>(stream), true);
}

fc_status fc_cache_update(fc_ctx *ctx, const fc_layer_desc *layer, const fc_kv_cache *kv,
                          const uint16_t *y_prev, uint16_t *y_cur, const int32_t *shift,
                          const uint8_t *reuse_mask, int32_t grid_w, int32_t B, void *stream) {
  if (!ctx) return fail(FC_ERR_INVALID_ARG, "fc_cache_update: null context");
  fc_status st = check_layer(ctx, layer, kv, B, "fc_cache_update");
  if (st != FC_OK) return st;
  if (!y_prev || !y_cur || !shift || !reuse_mask)
    return fail(FC_ERR_INVALID_ARG, "fc_cache_update: null buffer");
  if (kv->slot_map)
    return fail(FC_ERR_INVALID_ARG, "fc_cache_update: a slot-mapped cache is remapped once for all "
                "layers by fc_cache_update_layers");
  if (fc::overlap(y_prev, y_cur, (size_t)B * kv->frame_tokens * layer->d_model * 2))
    return fail(FC_ERR_INVALID_ARG, "fc_cache_update: y_prev and y_cur overlap");
  if (grid_w < 1 || kv->frame_tokens % grid_w)
    return fail(FC_ERR_SHAPE, "fc_cache_update: grid_w %d does not divide N=%d", grid_w,
                kv->frame_tokens);
  if ((layer->n_kv_heads * layer->head_dim) % 8 || layer->d_model % 8)
    return fail(FC_ERR_SHAPE, "fc_cache_update: row sizes must be multiples of 8 elements");
  st = use_device(ctx);
  if (st != FC_OK) return st;
  return fc::launch_cache_update(ctx, *layer, *kv, y_prev, y_cur, shift, reuse_mask, grid_w, B,
                                 reinterpret_cast<hipStream_t>(stream));
}

fc_status fc_cache_step(fc_ctx *ctx, const fc_layer_desc *layer, fc_kv_cache *kv,
                        const uint16_t *y_prev, uint16_t *y_cur, const int32_t *shift,
                        const uint8_t *reuse_mask, int32_t grid_w, int32_t flags, int32_t B,
                        void *stream) {
  if (!ctx) return fail(FC_ERR_INVALID_ARG, "fc_cache_step: null context");
  if (!kv) return fail(FC_ERR_INVALID_ARG, "fc_cache_step: null cache descriptor");
  if (flags <= 0 || (flags & ~(FC_ADVANCE_WINDOW | FC_REMAP)))
    return fail(FC_ERR_INVALID_ARG, "fc_cache_step: flags %d (FC_ADVANCE_WINDOW | FC_REMAP)", flags);
  if (kv->window < 1) return fail(FC_ERR_SHAPE, "fc_cache_step: window %d", kv->window);
  if (kv->head < 0 || kv->head >= kv->window)
    return fail(FC_ERR_INVALID_ARG, "fc_cache_step: head %d outside the window of %d frames",
                kv->head, kv->window);
  // the remap runs on the advanced layout; the caller's head changes only on success
  fc_kv_cache next = *kv;
  if (flags & FC_ADVANCE_WINDOW) next.head = (next.head + 1) % next.window;
  if (flags & FC_REMAP) {
    const fc_status st =
        fc_cache_update(ctx, layer, &next, y_prev, y_cur, shift, reuse_mask, grid_w, B, stream);
    if (st != FC_OK) return st;
  }
  kv->head = next.head;
  return FC_OK;
}

fc_status fc_cache_update_layers(fc_ctx *ctx, const fc_layer_desc *layer, int32_t n_layers,
                                 const fc_kv_cache *kvs, const uint16_t *const *y_prev,
                                 uint16_t *const *y_cur, const int32_t *shift,
                                 const uint8_t *reuse_mask, int32_t grid_w, int32_t B,
                                 void *stream) {
  if (!ctx) return fail(FC_ERR_INVALID_ARG, "fc_cache_update_layers: null context");
  if (n_layers < 1 || !kvs)
    return fail(FC_ERR_INVALID_ARG, "fc_cache_update_layers: n_layers %d or null cache array", n_layers);
  if ((y_prev == nullptr) != (y_cur == nullptr))
    return fail(FC_ERR_INVALID_ARG, "fc_cache_update_layers: y_prev and y_cur must both be given "
                "or both be NULL");
  if (!shift || !reuse_mask)
    return fail(FC_ERR_INVALID_ARG, "fc_cache_update_layers: null buffer");
  for (int l = 0; l < n_layers; ++l) {
    fc_status st = check_layer(ctx, layer, &kvs[l], B, "fc_cache_update_layers");
    if (st != FC_OK) return st;
    if (y_prev && (!y_prev[l] || !y_cur[l]))
      return fail(FC_ERR_INVALID_ARG, "fc_cache_update_layers: layer %d: null output buffer", l);
    if (kvs[l].text_tokens != kvs[0].text_tokens || kvs[l].frame_tokens != kvs[0].frame_tokens ||
        kvs[l].window != kvs[0].window || kvs[l].head != kvs[0].head ||
        kvs[l].trail_tokens != kvs[0].trail_tokens)
      return fail(FC_ERR_SHAPE, "fc_cache_update_layers: layer %d's cache layout or head differs", l);
    if (kvs[l].slot_map != kvs[0].slot_map)
      return fail(FC_ERR_INVALID_ARG, "fc_cache_update_layers: layer %d's slot map differs from "
                  "layer 0's (one map serves all layers)", l);
  }
  if (y_prev) {
    // one launch remaps every layer: no layer's output rows may overlap any layer's input
    // rows or another layer's output rows
    const size_t yb = (size_t)B * kvs[0].frame_tokens * layer->d_model * 2;
    for (int l = 0; l < n_layers; ++l)
      for (int m = 0; m < n_layers; ++m)
        if (fc::overlap(y_prev[l], y_cur[m], yb) || (m != l && fc::overlap(y_cur[l], y_cur[m], yb)))
          return fail(FC_ERR_INVALID_ARG, "fc_cache_update_layers: the output buffer of layer %d "
                      "overlaps an input or output buffer of layer %d", m, l);
  }
  if (grid_w < 1 || kvs[0].frame_tokens % grid_w)
    return fail(FC_ERR_SHAPE, "fc_cache_update_layers: grid_w %d does not divide N=%d", grid_w,
                kvs[0].frame_tokens);
  if ((layer->n_kv_heads * layer->head_dim) % 8 || layer->d_model % 8)
    return fail(FC_ERR_SHAPE, "fc_cache_update_layers: row sizes must be multiples of 8 elements");
  fc_status st = use_device(ctx);
  if (st != FC_OK) return st;
  return fc::launch_cache_update_layers(ctx, *layer, n_layers, kvs, y_prev, y_cur, shift, reuse_mask,
                                        grid_w, B, reinterpret_cast<hipStream_t>(stream));
}

static fc_status check_vit(fc_ctx *ctx, const fc_vit_desc *L, const fc_vit_cache *c, int B,
                           const char *who) {
  if (!ctx) return fail(FC_ERR_INVALID_ARG, "%s: null context", who);
  if (!L || !c) return fail(FC_ERR_INVALID_ARG, "%s: null layer or cache descriptor", who);
  if (!c->k || !c->v) return fail(FC_ERR_INVALID_ARG, "%s: null K or V cache", who);
  if (L->n_heads < 1 || L->head_dim < 16 || L->head_dim > 128 || L->head_dim % 16 ||
      (long)L->n_heads * L->head_dim != L->d_model)
    return fail(FC_ERR_INVALID_ARG, "%s: d_model %d must be n_heads %d x head_dim %d (head_dim a "
                "multiple of 16 up to 128)", who, L->d_model, L->n_heads, L->head_dim);
  if (L->d_model % fc::kGemmBK || L->d_model > 2048 || L->d_ffn < fc::kGemmBK ||
      L->d_ffn % fc::kGemmBK || L->d_ffn > (1 << 20))
    return fail(FC_ERR_SHAPE, "%s: d_model (<= 2048) and d_ffn must be multiples of %d", who,
                fc::kGemmBK);
  if (!(L->rms_eps > 0) || !(L->rope_theta > 1))
    return fail(FC_ERR_INVALID_ARG, "%s: rms_eps must be > 0 and rope_theta > 1", who);
  if (c->grid_h < 1 || c->grid_w < 1 || c->merge < 1 || c->merge > 4 || c->window < 0)
    return fail(FC_ERR_INVALID_ARG, "%s: grid %dx%d, merge %d, window %d", who, c->grid_h,
                c->grid_w, c->merge, c->window);
  if ((long)c->grid_h * c->merge > 128 || (long)c->grid_w * c->merge > 128)
    return fail(FC_ERR_UNSUPPORTED, "%s: patch grid sides up to 128", who);
  if (B < 1) return fail(FC_ERR_SHAPE, "%s: B=%d", who, B);
  const long N = (long)c->grid_h * c->grid_w;
  const long slots = (long)B * N * c->merge * c->merge;
  const fc_caps &cp = ctx->caps;
  const long rows = (long)cp.max_batch * cp.max_tokens;
  // the O reduction's sums of squares: one per slot and 1024-column chunk
  const long ssq_cap = rows * std::max<long>(8, (cp.max_d_model + 127) / 128);
  if (B > cp.max_batch || N > cp.max_tokens || slots * L->d_model > rows * cp.max_d_model ||
      slots * L->d_model > rows * cp.max_qkv || slots * L->d_ffn > rows * cp.max_ffn ||
      slots * ((L->d_model + 1023) / 1024) > ssq_cap)
    return fail(FC_ERR_CAPACITY, "%s: B=%d x %ld patches of d=%d, ffn=%d exceed the context's "
                "layer workspace", who, B, N * c->merge * c->merge, L->d_model, L->d_ffn);
  return FC_OK;
}

fc_status fc_vit_block_forward(fc_ctx *ctx, const fc_vit_desc *layer, const fc_vit_cache *cache,
                               const uint16_t *x, const int32_t *recompute_idx,
                               const int32_t *n_recompute, uint16_t *y, int32_t B, void *stream) {
  fc_status st = check_vit(ctx, layer, cache, B, "fc_vit_block_forward");
  if (st != FC_OK) return st;
  const fc_vit_desc &L = *layer;
  if (!x || !recompute_idx || !n_recompute || !y)
    return fail(FC_ERR_INVALID_ARG, "fc_vit_block_forward: null activation or index buffer");
  if (!L.w_qkv || !L.b_qkv || !L.w_o || !L.b_o || !L.w_gate_up || !L.b_gate_up || !L.w_down ||
      !L.b_down || !L.g1 || !L.g2)
    return fail(FC_ERR_INVALID_ARG, "fc_vit_block_forward: null weight pointer");
  if ((st = use_device(ctx)) != FC_OK) return st;
  return fc::launch_vit_block(ctx, L, *cache, x, recompute_idx, n_recompute, y, B,
                              reinterpret_cast<hipStream_t>(stream));
}

fc_status fc_vit_cache_update(fc_ctx *ctx, const fc_vit_desc *layer, const fc_vit_cache *cache,
                              const uint16_t *y_prev, uint16_t *y_cur, const int32_t *shift,
                              const uint8_t *reuse_mask, int32_t B, void *stream) {
  fc_status st = check_vit(ctx, layer, cache, B, "fc_vit_cache_update");
  if (st != FC_OK) return st;
  if (!shift || !reuse_mask || (!y_prev) != (!y_cur))
    return fail(FC_ERR_INVALID_ARG, "fc_vit_cache_update: null shift or reuse mask, or only one of "
                "y_prev and y_cur");
  const long mm = (long)cache->merge * cache->merge;
  const size_t rb = (size_t)B * cache->grid_h * cache->grid_w * mm * layer->d_model * 2;
  if (fc::overlap(y_prev, y_cur, rb))
    return fail(FC_ERR_INVALID_ARG, "fc_vit_cache_update: y_prev and y_cur overlap");
  if ((!cache->k_prev) != (!cache->v_prev) ||
      (cache->k_prev && (fc::overlap(cache->k_prev, cache->k, rb) || fc::overlap(cache->v_prev, cache->v, rb) ||
                         fc::overlap(cache->k_prev, cache->v, rb) || fc::overlap(cache->v_prev, cache->k, rb))))
    return fail(FC_ERR_INVALID_ARG, "fc_vit_cache_update: k_prev and v_prev must both be given, "
                "apart from k and v (no overlap), or both be NULL");
  // the in-place overwrite of the one frame slot stages the old K and V rows
  if (!cache->k_prev &&
      2L * B * cache->grid_h * cache->grid_w * mm * layer->d_model > (long)ctx->stage_elems)
    return fail(FC_ERR_CAPACITY, "fc_vit_cache_update: the frame's K/V rows exceed the context's "
                "staging buffer");
  if ((st = use_device(ctx)) != FC_OK) return st;
  return fc::launch_vit_cache_update(ctx, *layer, *cache, y_prev, y_cur, shift, reuse_mask, B,
                                     reinterpret_cast<hipStream_t>(stream));
}

fc_status fc_vit_merger_forward(fc_ctx *ctx, const fc_merger_desc *merger, const uint16_t *y,
                                const int32_t *recompute_idx, const int32_t *n_recompute,
                                uint16_t *x_out, int32_t n_tokens, int32_t B, void *stream) {
  const char *who = "fc_vit_merger_forward";
  if (!ctx) return fail(FC_ERR_INVALID_ARG, "%s: null context", who);
  if (!merger) return fail(FC_ERR_INVALID_ARG, "%s: null merger descriptor", who);
  const fc_merger_desc &M = *merger;
  if (!y || !recompute_idx || !n_recompute || !x_out)
    return fail(FC_ERR_INVALID_ARG, "%s: null activation or index buffer", who);
  if (!M.g || !M.w1 || !M.b1 || !M.w2 || !M.b2)
    return fail(FC_ERR_INVALID_ARG, "%s: null weight pointer", who);
  if (M.merge < 1 || M.merge > 4)
    return fail(FC_ERR_INVALID_ARG, "%s: merge %d (1 to 4)", who, M.merge);
  if (M.d_model < fc::kGemmBK || M.d_model % fc::kGemmBK || M.d_model > 2048 || M.d_out < 16 ||
      M.d_out % 16 || M.d_out > (1 << 16))
    return fail(FC_ERR_SHAPE, "%s: d_model %d (a multiple of %d up to 2048) and d_out %d (a "
                "multiple of 16)", who, M.d_model, fc::kGemmBK, M.d_out);
  if (!(M.rms_eps > 0)) return fail(FC_ERR_INVALID_ARG, "%s: rms_eps must be > 0", who);
  if (B < 1 || n_tokens < 1) return fail(FC_ERR_SHAPE, "%s: B=%d, n_tokens=%d", who, B, n_tokens);
  const fc_caps &cp = ctx->caps;
  const long hidden = (long)M.merge * M.merge * M.d_model;
  const long rows = (long)cp.max_batch * cp.max_tokens;
  if (B > cp.max_batch || n_tokens > cp.max_tokens || 2L * B * n_tokens * hidden > rows * cp.max_ffn)
    return fail(FC_ERR_CAPACITY, "%s: B=%d x %d tokens of %ld merged features exceed the "
                "context's MLP workspace", who, B, n_tokens, hidden);
  fc_status st = use_device(ctx);
  if (st != FC_OK) return st;
  return fc::launch_vit_merger(ctx, M, y, recompute_idx, n_recompute, x_out, n_tokens, B,
                               reinterpret_cast<hipStream_t>(stream));
}

size_t fc_slot_state_bytes(int32_t B, int32_t S) { return fc::slot_state_bytes(B, S); }

fc_status fc_slot_map_init(fc_ctx *ctx, const fc_layer_desc *layer, const fc_kv_cache *kv,
                           int32_t B, void *stream) {
  if (!ctx) return fail(FC_ERR_INVALID_ARG, "fc_slot_map_init: null context");
  fc_status st = check_layer(ctx, layer, kv, B, "fc_slot_map_init");
  if (st != FC_OK) return st;
  if (!kv->slot_map) return fail(FC_ERR_INVALID_ARG, "fc_slot_map_init: the cache has no slot map");
  if (kv->frame_tokens > fc::kMaxTokens)
    return fail(FC_ERR_UNSUPPORTED, "fc_slot_map_init: N=%d > %d", kv->frame_tokens, fc::kMaxTokens);
  if ((st = use_device(ctx)) != FC_OK) return st;
  return fc::launch_slot_init(ctx, *kv, B, reinterpret_cast<hipStream_t>(stream));
}

int32_t fc_debug(int32_t on) {
  const int prev = fc::g_debug.load();
  if (on >= 0) fc::g_debug.store(on != 0 ? 1 : 0);
  return prev;
}

fc_status fc_profile_enable(fc_ctx *ctx, int32_t on) {
  if (!ctx) return fail(FC_ERR_INVALID_ARG, "fc_profile_enable: null context");
  ctx->prof = on != 0;
  return FC_OK;
}

fc_status fc_profile_only(fc_ctx *ctx, const char *name) {
  if (!ctx) return fail(FC_ERR_INVALID_ARG, "fc_profile_only: null context");
  ctx->prof_only = name ? name : "";
  return FC_OK;
}

fc_status fc_profile_read(fc_ctx *ctx, const char *name, double *total_ms, int64_t *launches,
                          int32_t reset) {
  if (!ctx) return fail(FC_ERR_INVALID_ARG, "fc_profile_read: null context");
  double tot = 0.0;
  int64_t cnt = 0;
  for (auto &r : ctx->recs) {
    if (name && std::strcmp(name, r.name) != 0) continue;
    hipError_t e = hipEventSynchronize(r.stop);
    if (e != hipSuccess) return fail(FC_ERR_HIP, "hipEventSynchronize: %s", hipGetErrorString(e));
    float ms = 0.f;
    e = hipEventElapsedTime(&ms, r.start, r.stop);
    if (e != hipSuccess) return fail(FC_ERR_HIP, "hipEventElapsedTime: %s", hipGetErrorString(e));
    tot += ms;
    ++cnt;
  }
  if (total_ms) *total_ms = tot;
  if (launches) *launches = cnt;
  if (reset) {
    for (auto &r : ctx->recs) {
      hipEventSynchronize(r.stop);
      ctx->pool.push_back(r.start);
      ctx->pool.push_back(r.stop);
    }
    ctx->recs.clear();
  }
  return FC_OK;
}

}  // extern "C"
