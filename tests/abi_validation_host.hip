// Host-side driver over the argument validation of the C ABI, built together with the
// library sources with the host code under AddressSanitizer and UndefinedBehaviorSanitizer
// (tests/test_abi_sanitize.py) and run on a machine without a GPU.  A context is built by
// hand (caps set, no device buffers), so every check of fc_select, fc_select_carry,
// fc_select_noalloc, fc_phase_correlate, fc_layer_forward, fc_layer_forward_trail, fc_cache_update and
// fc_cache_update_layers runs, down to the first device call, which then fails cleanly.
// Extreme sizes probe the overflow of the size arithmetic.  Exit status 0: every
// expectation held (the sanitizers abort on a finding).
#include <climits>
#include <cstdio>
#include <cstring>

#include "../paper_2604_24391_amd/csrc/fc_internal.h"

static int g_fail = 0;

#define EXPECT(call, want)                                                              \
  do {                                                                                  \
    const fc_status _s = (call);                                                        \
    const char *_m = fc_last_error();                                                   \
    if (_s != (want) || (_s != FC_OK && (!_m || !*_m || std::strlen(_m) >= 1024))) {    \
      std::printf("FAIL line %d: %s -> %d (want %d): %s\n", __LINE__, #call, (int)_s,  \
                  (int)(want), _m ? _m : "(null)");                                     \
      ++g_fail;                                                                         \
    }                                                                                   \
  } while (0)

// any status but OK: calls that pass validation stop at the first device call
#define EXPECT_DEVICE_FAIL(call)                                                        \
  do {                                                                                  \
    const fc_status _s = (call);                                                        \
    if (_s != FC_ERR_HIP && _s != FC_ERR_NO_DEVICE) {                                   \
      std::printf("FAIL line %d: %s -> %d (want a device error): %s\n", __LINE__, #call, \
                  (int)_s, fc_last_error());                                            \
      ++g_fail;                                                                         \
    }                                                                                   \
  } while (0)

static fc_select_params default_params() {
  fc_select_params p{};
  p.patch = 14;
  p.merge = 2;
  p.tau_mig = 0.12;
  p.lambda_ = 0.25;
  p.alpha_min = 0.08;
  p.alpha_max = 0.5;
  p.adaptive = 1;
  p.alpha_fixed = 0.5;
  p.entropy_norm = 1;
  return p;
}

static fc_layer_desc qwen_layer(uint16_t *w) {
  fc_layer_desc L{};
  L.d_model = 3584;
  L.n_heads = 28;
  L.n_kv_heads = 4;
  L.head_dim = 128;
  L.d_ffn = 18944;
  L.rms_eps = 1e-6f;
  L.rope_theta = 1e6;
  L.w_qkv = L.b_qkv = L.w_o = L.w_gate = L.w_up = L.w_down = L.g_attn = L.g_mlp = w;
  return L;
}

static fc_kv_cache qwen_cache(uint16_t *k, uint16_t *v) {
  fc_kv_cache c{};
  c.k = k;
  c.v = v;
  c.text_tokens = 128;
  c.frame_tokens = 256;
  c.window = 8;
  c.head = 0;
  return c;
}

int main() {
  // buffers are never dereferenced on the host: any non-null address will do
  alignas(16) static unsigned char host[4096];
  float *f = reinterpret_cast<float *>(host);
  uint16_t *h16 = reinterpret_cast<uint16_t *>(host);
  int32_t *i32 = reinterpret_cast<int32_t *>(host);
  uint8_t *u8 = host;
  // buffers that a remap reads and writes at once must not overlap: stand-ins for
  // distinct allocations, 1 TiB apart (never dereferenced either)
  auto far16 = [](int i) { return reinterpret_cast<uint16_t *>((uintptr_t)(i + 1) << 40); };

  fc_select_out out{};
  out.sim = f;
  out.energy = reinterpret_cast<double *>(host);
  out.reuse_mask = u8;
  out.recompute_idx = i32;
  out.n_recompute = i32;
  out.shift = i32;
  out.scalars = reinterpret_cast<double *>(host);
  out.counts = i32;

  // ---------------------------------------------------------------- context-free calls
  EXPECT(fc_create(nullptr, 0, nullptr), FC_ERR_INVALID_ARG);
  EXPECT(fc_destroy(nullptr), FC_ERR_INVALID_ARG);
  if (!fc_version() || !*fc_version()) { std::printf("FAIL: empty version\n"); ++g_fail; }
  if (fc_select_state_bytes(-1, 448, 448) != 0 || fc_select_state_bytes(1, 0, 448) != 0 ||
      fc_select_state_bytes(1, 448, INT_MIN) != 0) {
    std::printf("FAIL: state bytes of invalid sizes must be 0\n");
    ++g_fail;
  }
  (void)fc_select_state_bytes(INT_MAX, INT_MAX, INT_MAX);    // no overflow UB
  (void)fc_select_state_bytes(INT_MAX, 14, 14);
  const fc_select_params p = default_params();
  EXPECT(fc_select_noalloc(nullptr, f, f, 1, 448, 448, &out, nullptr), FC_ERR_INVALID_ARG);
  EXPECT(fc_select_noalloc(&p, f, f, INT_MAX, 448, 448, &out, nullptr), FC_ERR_CAPACITY);
  EXPECT(fc_select_noalloc(&p, f, f, 1, INT_MAX - INT_MAX % 28, 28, &out, nullptr),
         FC_ERR_UNSUPPORTED);
  EXPECT(fc_select_noalloc(&p, f, f, 64, 448, 448, &out, nullptr), FC_ERR_CAPACITY);
  EXPECT_DEVICE_FAIL(fc_select_noalloc(&p, f, f, 1, 224, 224, &out, nullptr));
  {
    fc_select_params q = p;
    q.patch = 16;
    EXPECT(fc_select_noalloc(&q, f, f, 1, 448, 448, &out, nullptr), FC_ERR_UNSUPPORTED);
    q = p;
    q.merge = INT_MAX;
    EXPECT(fc_select_noalloc(&q, f, f, 1, 448, 448, &out, nullptr), FC_ERR_INVALID_ARG);
    q = p;
    q.tau_sim = __builtin_nan("");
    EXPECT(fc_select_noalloc(&q, f, f, 1, 448, 448, &out, nullptr), FC_ERR_INVALID_ARG);
    q = p;
    q.alpha_min = 0.95;
    EXPECT(fc_select_noalloc(&q, f, f, 1, 448, 448, &out, nullptr), FC_ERR_INVALID_ARG);
    q = p;
    q.no_align = 2;
    EXPECT(fc_select_noalloc(&q, f, f, 1, 448, 448, &out, nullptr), FC_ERR_INVALID_ARG);
    fc_select_out o2 = out;
    o2.counts = nullptr;
    EXPECT(fc_select_noalloc(&p, f, f, 1, 448, 448, &o2, nullptr), FC_ERR_INVALID_ARG);
    EXPECT(fc_select_noalloc(&p, f, f, 1, 450, 448, &out, nullptr), FC_ERR_SHAPE);
    EXPECT(fc_select_noalloc(&p, f, f, 0, 448, 448, &out, nullptr), FC_ERR_SHAPE);
    EXPECT(fc_select_noalloc(&p, f, f, 1, 28 * 64, 28 * 64, &out, nullptr), FC_ERR_UNSUPPORTED);
    q = p;
    q.align_pixel = 2;
    EXPECT(fc_select_noalloc(&q, f, f, 1, 448, 448, &out, nullptr), FC_ERR_INVALID_ARG);
    q.align_pixel = 1;
    EXPECT(fc_select_noalloc(&q, f, f, 1, 420, 448, &out, nullptr), FC_ERR_UNSUPPORTED);
    EXPECT(fc_select_noalloc(&q, f, f, 8, 448, 448, &out, nullptr), FC_ERR_CAPACITY);
    EXPECT_DEVICE_FAIL(fc_select_noalloc(&q, f, f, 1, 448, 448, &out, nullptr));
  }
  if (fc_debug(-1) != 0 && fc_debug(-1) != 1) { std::printf("FAIL: debug mode\n"); ++g_fail; }

  // --------------------------------------------- a context by hand: caps, no device memory
  fc_ctx *ctx = new fc_ctx;
  ctx->device = 0;
  ctx->caps.max_batch = 4;
  ctx->caps.max_height = 448;
  ctx->caps.max_width = 448;
  ctx->caps.max_tokens = 256;
  ctx->caps.max_seq = 128 + 8 * 256 + 64;
  ctx->caps.max_d_model = 3584;
  ctx->caps.max_ffn = 18944;
  ctx->caps.max_qkv = 4608;
  ctx->stage_elems = (size_t)4 * 256 * 4608;      // as fc_create sizes it for these caps

  EXPECT(fc_select(nullptr, &p, f, f, 1, 448, 448, &out, nullptr), FC_ERR_INVALID_ARG);
  EXPECT(fc_select(ctx, &p, f, f, 5, 448, 448, &out, nullptr), FC_ERR_CAPACITY);
  EXPECT(fc_select(ctx, &p, f, f, 1, 896, 448, &out, nullptr), FC_ERR_CAPACITY);
  EXPECT_DEVICE_FAIL(fc_select(ctx, &p, f, f, 4, 448, 448, &out, nullptr));
  EXPECT(fc_select_carry(ctx, &p, host, f, host, 1, 448, 448, &out, nullptr), FC_ERR_INVALID_ARG);
  EXPECT(fc_select_carry(ctx, &p, host, f, host + 64, 1, 448, 448, &out, nullptr), FC_ERR_INVALID_ARG);
  EXPECT_DEVICE_FAIL(fc_select_carry(ctx, &p, reinterpret_cast<unsigned char *>(far16(5)), f, host, 1,
                                     448, 448, &out, nullptr));
  EXPECT(fc_select_carry(ctx, &p, nullptr, f, nullptr, 1, 448, 448, &out, nullptr),
         FC_ERR_INVALID_ARG);
  EXPECT(fc_select_carry(ctx, &p, nullptr, f, host, INT_MAX, 448, 448, &out, nullptr),
         FC_ERR_CAPACITY);
  EXPECT_DEVICE_FAIL(fc_select_carry(ctx, &p, nullptr, f, host, 1, 448, 448, &out, nullptr));
  {
    fc_select_params q = p;
    q.align_pixel = 1;
    EXPECT(fc_select_carry(ctx, &q, nullptr, f, host, 1, 448, 448, &out, nullptr),
           FC_ERR_UNSUPPORTED);
    EXPECT_DEVICE_FAIL(fc_select(ctx, &q, f, f, 1, 448, 448, &out, nullptr));
    double *sp = reinterpret_cast<double *>(host);
    EXPECT(fc_phase_correlate(nullptr, f, f, 1, 448, 448, sp, nullptr, nullptr, nullptr),
           FC_ERR_INVALID_ARG);
    EXPECT(fc_phase_correlate(ctx, f, f, 1, 448, 448, nullptr, nullptr, nullptr, nullptr),
           FC_ERR_INVALID_ARG);
    EXPECT(fc_phase_correlate(ctx, f, f, 1, 448, 420, sp, nullptr, nullptr, nullptr),
           FC_ERR_UNSUPPORTED);
    EXPECT(fc_phase_correlate(ctx, f, f, 1, 7 * 256, 448, sp, nullptr, nullptr, nullptr),
           FC_ERR_UNSUPPORTED);
    EXPECT(fc_phase_correlate(ctx, f, f, 1, INT_MAX, 448, sp, nullptr, nullptr, nullptr),
           FC_ERR_UNSUPPORTED);
    EXPECT(fc_phase_correlate(ctx, f, f, 0, 448, 448, sp, nullptr, nullptr, nullptr), FC_ERR_SHAPE);
    EXPECT(fc_phase_correlate(ctx, f, f, 5, 448, 448, sp, nullptr, nullptr, nullptr),
           FC_ERR_CAPACITY);
    EXPECT(fc_phase_correlate(ctx, f, f, 1, 896, 448, sp, nullptr, nullptr, nullptr),
           FC_ERR_CAPACITY);
    EXPECT_DEVICE_FAIL(fc_phase_correlate(ctx, nullptr, f, 4, 448, 448, sp, nullptr, nullptr,
                                          nullptr));
    EXPECT(fc_phase_correlate_rotation(nullptr, f, f, 1, 448, 448, sp, sp, nullptr),
           FC_ERR_INVALID_ARG);
    EXPECT(fc_phase_correlate_rotation(ctx, f, f, 1, 14, 448, sp, sp, nullptr), FC_ERR_UNSUPPORTED);
    EXPECT(fc_phase_correlate_rotation(ctx, f, f, 1, 448, 448, sp, nullptr, nullptr),
           FC_ERR_INVALID_ARG);
    EXPECT(fc_phase_correlate_rotation(ctx, f, f, 5, 448, 448, sp, sp, nullptr), FC_ERR_CAPACITY);
    EXPECT_DEVICE_FAIL(fc_phase_correlate_rotation(ctx, f, f, 2, 448, 224, nullptr, sp, nullptr));
    q.align_rotation = 1;
    EXPECT_DEVICE_FAIL(fc_select(ctx, &q, f, f, 1, 448, 448, &out, nullptr));
    q.align_pixel = 0;
    EXPECT(fc_select(ctx, &q, f, f, 1, 448, 448, &out, nullptr), FC_ERR_INVALID_ARG);
    q.align_pixel = 1;
    q.align_rotation = 2;
    EXPECT(fc_select(ctx, &q, f, f, 1, 448, 448, &out, nullptr), FC_ERR_INVALID_ARG);
  }

  fc_layer_desc L = qwen_layer(h16);
  fc_kv_cache kv = qwen_cache(h16, h16);
  auto fwd = [&](const fc_layer_desc &l, const fc_kv_cache &c, int B) {
    return fc_layer_forward(ctx, &l, &c, h16, i32, i32, h16, B, nullptr);
  };
  EXPECT(fc_layer_forward(nullptr, &L, &kv, h16, i32, i32, h16, 1, nullptr), FC_ERR_INVALID_ARG);
  EXPECT(fc_layer_forward(ctx, nullptr, &kv, h16, i32, i32, h16, 1, nullptr), FC_ERR_INVALID_ARG);
  EXPECT(fc_layer_forward(ctx, &L, &kv, nullptr, i32, i32, h16, 1, nullptr), FC_ERR_INVALID_ARG);
  EXPECT_DEVICE_FAIL(fwd(L, kv, 1));
  EXPECT(fwd(L, kv, 0), FC_ERR_SHAPE);
  EXPECT(fwd(L, kv, 5), FC_ERR_CAPACITY);
  EXPECT(fwd(L, kv, INT_MAX), FC_ERR_CAPACITY);
  {
    fc_layer_desc l = L;
    l.head_dim = INT_MAX;                      // products of dimensions must not overflow
    EXPECT(fwd(l, kv, 1), FC_ERR_UNSUPPORTED);
    l = L;
    l.d_ffn = INT_MAX - 1;
    EXPECT(fwd(l, kv, 1), FC_ERR_SHAPE);
    l.d_ffn = INT_MAX - INT_MAX % 64;
    EXPECT(fwd(l, kv, 1), FC_ERR_CAPACITY);
    l = L;
    l.n_kv_heads = 3;
    EXPECT(fwd(l, kv, 1), FC_ERR_SHAPE);
    l = L;
    l.n_heads = 0;
    EXPECT(fwd(l, kv, 1), FC_ERR_INVALID_ARG);
    l = L;
    l.d_model = 8256;
    EXPECT(fwd(l, kv, 1), FC_ERR_UNSUPPORTED);
    l = L;
    l.rms_eps = 0.f;
    EXPECT(fwd(l, kv, 1), FC_ERR_INVALID_ARG);
    l = L;
    l.rope_theta = __builtin_nan("");
    EXPECT(fwd(l, kv, 1), FC_ERR_INVALID_ARG);
    l = L;
    l.w_down = nullptr;
    EXPECT(fwd(l, kv, 1), FC_ERR_INVALID_ARG);
    l = L;
    l.n_heads = 32;                            // 8 query heads per KV head: not built
    l.d_model = 3584;
    ctx->caps.max_qkv = 8192;
    EXPECT(fwd(l, kv, 1), FC_ERR_UNSUPPORTED);
    ctx->caps.max_qkv = 4608;
  }
  {
    fc_kv_cache c = kv;
    c.head = 8;
    EXPECT(fwd(L, c, 1), FC_ERR_INVALID_ARG);
    c = kv;
    c.window = INT_MAX;                        // T + W N must not overflow
    c.frame_tokens = INT_MAX;
    EXPECT(fwd(L, c, 1), FC_ERR_CAPACITY);
    c = kv;
    c.trail_tokens = -1;
    EXPECT(fwd(L, c, 1), FC_ERR_INVALID_ARG);
    c = kv;
    c.trail_tokens = INT_MAX;
    EXPECT(fwd(L, c, 1), FC_ERR_CAPACITY);
    c = kv;
    c.k = nullptr;
    EXPECT(fwd(L, c, 1), FC_ERR_INVALID_ARG);
    c = kv;
    c.mrope_section[0] = 16;
    c.mrope_section[1] = 24;
    c.mrope_section[2] = 24;
    c.grid_w = 16;
    EXPECT_DEVICE_FAIL(fwd(L, c, 1));
    c.grid_w = 15;
    EXPECT(fwd(L, c, 1), FC_ERR_SHAPE);
    c.grid_w = 0;
    EXPECT(fwd(L, c, 1), FC_ERR_SHAPE);
    c.grid_w = 16;
    c.mrope_section[2] = INT_MAX;              // the sum must not overflow
    EXPECT(fwd(L, c, 1), FC_ERR_INVALID_ARG);
    c.mrope_section[2] = 20;
    EXPECT(fwd(L, c, 1), FC_ERR_INVALID_ARG);
    c.mrope_section[0] = -8;
    c.mrope_section[2] = 40;
    EXPECT(fwd(L, c, 1), FC_ERR_INVALID_ARG);
    c = kv;
    c.trail_tokens = 64;
    EXPECT_DEVICE_FAIL(fc_layer_forward_trail(ctx, &L, &c, h16, h16, 1, nullptr));
    EXPECT(fc_layer_forward_trail(ctx, &L, &kv, h16, h16, 1, nullptr), FC_ERR_INVALID_ARG);
    EXPECT(fc_layer_forward_trail(ctx, &L, &c, nullptr, h16, 1, nullptr), FC_ERR_INVALID_ARG);
    c.trail_tokens = 65;
    EXPECT(fc_layer_forward_trail(ctx, &L, &c, h16, h16, 1, nullptr), FC_ERR_CAPACITY);
  }
  {
    uint16_t *y2 = far16(0);
    EXPECT(fc_cache_update(ctx, &L, &kv, h16, h16, i32, u8, 16, 1, nullptr), FC_ERR_INVALID_ARG);
    // a partial overlap: 8 elements apart
    EXPECT(fc_cache_update(ctx, &L, &kv, h16, h16 + 8, i32, u8, 16, 1, nullptr), FC_ERR_INVALID_ARG);
    EXPECT(fc_cache_update(ctx, &L, &kv, h16, y2, i32, u8, 15, 1, nullptr), FC_ERR_SHAPE);
    EXPECT(fc_cache_update(ctx, &L, &kv, h16, y2, nullptr, u8, 16, 1, nullptr), FC_ERR_INVALID_ARG);
    {
      fc_kv_cache ks = kv;
      const int h0 = ks.head;
      EXPECT(fc_cache_step(ctx, &L, &ks, h16, y2, i32, u8, 16, 0, 1, nullptr), FC_ERR_INVALID_ARG);
      EXPECT(fc_cache_step(ctx, &L, &ks, h16, y2, i32, u8, 16, 4, 1, nullptr), FC_ERR_INVALID_ARG);
      EXPECT(fc_cache_step(nullptr, &L, &ks, h16, y2, i32, u8, 16, FC_REMAP, 1, nullptr), FC_ERR_INVALID_ARG);
      EXPECT(fc_cache_step(ctx, &L, nullptr, h16, y2, i32, u8, 16, FC_REMAP, 1, nullptr), FC_ERR_INVALID_ARG);
      EXPECT(fc_cache_step(ctx, &L, &ks, nullptr, nullptr, nullptr, nullptr, 16, FC_ADVANCE_WINDOW, 1, nullptr), FC_OK);
      if (ks.head != (h0 + 1) % ks.window) {
        std::printf("FAIL: fc_cache_step did not advance the head\n");
        ++g_fail;
      }
      const int h1 = ks.head;
      EXPECT(fc_cache_step(ctx, &L, &ks, h16, y2, nullptr, u8, 16, FC_ADVANCE_WINDOW | FC_REMAP, 1, nullptr),
             FC_ERR_INVALID_ARG);
      if (ks.head != h1) {
        std::printf("FAIL: a failing fc_cache_step moved the head\n");
        ++g_fail;
      }
      {
        fc_kv_cache kb = ks;
        kb.head = kb.window;
        EXPECT(fc_cache_step(ctx, &L, &kb, nullptr, nullptr, nullptr, nullptr, 16, FC_ADVANCE_WINDOW, 1,
                             nullptr),
               FC_ERR_INVALID_ARG);
      }
      EXPECT_DEVICE_FAIL(fc_cache_step(ctx, &L, &ks, h16, y2, i32, u8, 16, FC_REMAP, 1, nullptr));
    }
    EXPECT_DEVICE_FAIL(fc_cache_update(ctx, &L, &kv, h16, y2, i32, u8, 16, 1, nullptr));
    fc_kv_cache kvs[3] = {kv, kv, kv};
    const uint16_t *yp[3] = {h16, h16, h16};
    uint16_t *yc[3] = {far16(1), far16(2), far16(3)};
    EXPECT_DEVICE_FAIL(fc_cache_update_layers(ctx, &L, 3, kvs, yp, yc, i32, u8, 16, 1, nullptr));
    yc[2] = yc[1] + 8;                 // two layers' outputs overlap
    EXPECT(fc_cache_update_layers(ctx, &L, 3, kvs, yp, yc, i32, u8, 16, 1, nullptr),
           FC_ERR_INVALID_ARG);
    yc[2] = far16(3);
    EXPECT(fc_cache_update_layers(ctx, &L, 0, kvs, yp, yc, i32, u8, 16, 1, nullptr),
           FC_ERR_INVALID_ARG);
    EXPECT(fc_cache_update_layers(ctx, &L, INT_MIN, kvs, yp, yc, i32, u8, 16, 1, nullptr),
           FC_ERR_INVALID_ARG);
    kvs[2].head = 1;
    EXPECT(fc_cache_update_layers(ctx, &L, 3, kvs, yp, yc, i32, u8, 16, 1, nullptr), FC_ERR_SHAPE);
    kvs[2] = kv;
    yc[1] = h16;
    EXPECT(fc_cache_update_layers(ctx, &L, 3, kvs, yp, yc, i32, u8, 16, 1, nullptr),
           FC_ERR_INVALID_ARG);
  }
  {
    // slot-mapped caches
    int32_t *smap = i32;
    fc_kv_cache mk = kv;
    mk.slot_map = smap;
    uint16_t *y2 = far16(0);
    EXPECT(fc_cache_update(ctx, &L, &mk, h16, y2, i32, u8, 16, 1, nullptr), FC_ERR_INVALID_ARG);
    fc_kv_cache kvs[2] = {mk, mk};
    const uint16_t *yp[2] = {h16, h16};
    uint16_t *yc[2] = {far16(1), far16(2)};
    EXPECT_DEVICE_FAIL(fc_cache_update_layers(ctx, &L, 2, kvs, yp, yc, i32, u8, 16, 1, nullptr));
    EXPECT_DEVICE_FAIL(fc_cache_update_layers(ctx, &L, 2, kvs, nullptr, nullptr, i32, u8, 16, 1,
                                              nullptr));
    EXPECT(fc_cache_update_layers(ctx, &L, 2, kvs, yp, nullptr, i32, u8, 16, 1, nullptr),
           FC_ERR_INVALID_ARG);
    kvs[1].slot_map = nullptr;
    EXPECT(fc_cache_update_layers(ctx, &L, 2, kvs, yp, yc, i32, u8, 16, 1, nullptr),
           FC_ERR_INVALID_ARG);
    kvs[1] = mk;
    kvs[1].trail_tokens = 8;
    EXPECT(fc_cache_update_layers(ctx, &L, 2, kvs, yp, yc, i32, u8, 16, 1, nullptr), FC_ERR_SHAPE);
    EXPECT(fc_slot_map_init(ctx, &L, &kv, 1, nullptr), FC_ERR_INVALID_ARG);
    EXPECT(fc_slot_map_init(nullptr, &L, &mk, 1, nullptr), FC_ERR_INVALID_ARG);
    EXPECT(fc_slot_map_init(ctx, &L, &mk, 0, nullptr), FC_ERR_SHAPE);
    EXPECT_DEVICE_FAIL(fc_slot_map_init(ctx, &L, &mk, 1, nullptr));
    EXPECT_DEVICE_FAIL(fwd(L, mk, 1));
    if (fc_slot_state_bytes(0, 10) != 0 || fc_slot_state_bytes(1, -1) != 0 ||
        fc_slot_state_bytes(2, 100) != (3 * 2 * 100 + 2) * 4) {
      std::printf("FAIL: slot state bytes\n");
      ++g_fail;
    }
    (void)fc_slot_state_bytes(INT_MAX, INT_MAX);
  }
  {
    // vision block
    fc_vit_desc vd{};
    vd.d_model = 1280;
    vd.n_heads = 16;
    vd.head_dim = 80;
    vd.d_ffn = 3456;
    vd.rms_eps = 1e-6f;
    vd.rope_theta = 1e4;
    vd.w_qkv = vd.b_qkv = vd.w_o = vd.b_o = vd.w_gate_up = vd.b_gate_up = vd.w_down = vd.b_down =
        vd.g1 = vd.g2 = h16;
    fc_vit_cache vc{};
    vc.k = vc.v = h16;
    vc.grid_h = vc.grid_w = 16;
    vc.merge = 2;
    vc.window = 4;
    auto vfwd = [&](const fc_vit_desc &l, const fc_vit_cache &c, int B) {
      return fc_vit_block_forward(ctx, &l, &c, h16, i32, i32, h16, B, nullptr);
    };
    EXPECT_DEVICE_FAIL(vfwd(vd, vc, 1));
    EXPECT(fc_vit_block_forward(nullptr, &vd, &vc, h16, i32, i32, h16, 1, nullptr), FC_ERR_INVALID_ARG);
    EXPECT(fc_vit_block_forward(ctx, &vd, &vc, nullptr, i32, i32, h16, 1, nullptr), FC_ERR_INVALID_ARG);
    EXPECT(vfwd(vd, vc, 0), FC_ERR_SHAPE);
    EXPECT(vfwd(vd, vc, 5), FC_ERR_CAPACITY);
    fc_vit_desc l2 = vd;
    l2.head_dim = 81;
    EXPECT(vfwd(l2, vc, 1), FC_ERR_INVALID_ARG);
    l2.head_dim = 40;                  // a multiple of 8 but not of 16
    l2.n_heads = 32;
    EXPECT(vfwd(l2, vc, 1), FC_ERR_INVALID_ARG);
    l2 = vd;
    l2.n_heads = INT_MAX;
    EXPECT(vfwd(l2, vc, 1), FC_ERR_INVALID_ARG);
    l2 = vd;
    l2.d_ffn = 3420;
    EXPECT(vfwd(l2, vc, 1), FC_ERR_SHAPE);
    l2 = vd;
    l2.w_down = nullptr;
    EXPECT(vfwd(l2, vc, 1), FC_ERR_INVALID_ARG);
    fc_vit_cache c2 = vc;
    c2.grid_h = 65;
    EXPECT(vfwd(vd, c2, 1), FC_ERR_UNSUPPORTED);
    c2 = vc;
    c2.grid_h = c2.grid_w = INT_MAX;
    EXPECT(vfwd(vd, c2, 1), FC_ERR_UNSUPPORTED);
    c2 = vc;
    c2.window = -1;
    EXPECT(vfwd(vd, c2, 1), FC_ERR_INVALID_ARG);
    c2 = vc;
    c2.k = nullptr;
    EXPECT(vfwd(vd, c2, 1), FC_ERR_INVALID_ARG);
    uint16_t *y2 = far16(0);
    EXPECT_DEVICE_FAIL(fc_vit_cache_update(ctx, &vd, &vc, h16, y2, i32, u8, 1, nullptr));
    EXPECT(fc_vit_cache_update(ctx, &vd, &vc, h16, h16 + 8, i32, u8, 1, nullptr), FC_ERR_INVALID_ARG);
    EXPECT(fc_vit_cache_update(ctx, &vd, &vc, h16, h16, i32, u8, 1, nullptr), FC_ERR_INVALID_ARG);
    EXPECT(fc_vit_cache_update(ctx, &vd, &vc, h16, y2, nullptr, u8, 1, nullptr), FC_ERR_INVALID_ARG);
    EXPECT(fc_vit_cache_update(ctx, &vd, &vc, h16, nullptr, i32, u8, 1, nullptr), FC_ERR_INVALID_ARG);
    EXPECT_DEVICE_FAIL(fc_vit_cache_update(ctx, &vd, &vc, nullptr, nullptr, i32, u8, 1, nullptr));
    fc_vit_cache c3 = vc;
    c3.k_prev = y2;                    // k_prev without v_prev
    EXPECT(fc_vit_cache_update(ctx, &vd, &c3, nullptr, nullptr, i32, u8, 1, nullptr), FC_ERR_INVALID_ARG);
    c3.v_prev = h16;                   // v_prev is v itself
    EXPECT(fc_vit_cache_update(ctx, &vd, &c3, nullptr, nullptr, i32, u8, 1, nullptr), FC_ERR_INVALID_ARG);
    c3.v_prev = h16 + 64;              // v_prev overlaps v in part
    EXPECT(fc_vit_cache_update(ctx, &vd, &c3, nullptr, nullptr, i32, u8, 1, nullptr), FC_ERR_INVALID_ARG);
    c3.v_prev = y2;
    EXPECT_DEVICE_FAIL(fc_vit_cache_update(ctx, &vd, &c3, nullptr, nullptr, i32, u8, 1, nullptr));
    // separate buffers need no staging: with a one-element staging buffer only the
    // in-place remap is refused
    fc_vit_cache c4 = vc;
    const size_t stage_keep = ctx->stage_elems;
    ctx->stage_elems = 1;
    EXPECT(fc_vit_cache_update(ctx, &vd, &c4, nullptr, nullptr, i32, u8, 1, nullptr), FC_ERR_CAPACITY);
    EXPECT_DEVICE_FAIL(fc_vit_cache_update(ctx, &vd, &c3, nullptr, nullptr, i32, u8, 1, nullptr));
    ctx->stage_elems = stage_keep;
  }
  {
    // patch merger
    fc_merger_desc md{};
    md.d_model = 1280;
    md.merge = 2;
    md.d_out = 3584;
    md.rms_eps = 1e-6f;
    md.g = md.w1 = md.b1 = md.w2 = md.b2 = h16;
    auto mfwd = [&](const fc_merger_desc &m, int n, int B) {
      return fc_vit_merger_forward(ctx, &m, h16, i32, i32, h16, n, B, nullptr);
    };
    EXPECT_DEVICE_FAIL(mfwd(md, 256, 4));
    EXPECT(fc_vit_merger_forward(nullptr, &md, h16, i32, i32, h16, 256, 1, nullptr), FC_ERR_INVALID_ARG);
    EXPECT(fc_vit_merger_forward(ctx, nullptr, h16, i32, i32, h16, 256, 1, nullptr), FC_ERR_INVALID_ARG);
    EXPECT(fc_vit_merger_forward(ctx, &md, h16, nullptr, i32, h16, 256, 1, nullptr), FC_ERR_INVALID_ARG);
    EXPECT(mfwd(md, 256, 0), FC_ERR_SHAPE);
    EXPECT(mfwd(md, 0, 1), FC_ERR_SHAPE);
    EXPECT(mfwd(md, 256, 5), FC_ERR_CAPACITY);
    EXPECT(mfwd(md, 257, 1), FC_ERR_CAPACITY);
    fc_merger_desc m2 = md;
    m2.merge = 4;
    m2.d_model = 2048;
    EXPECT(mfwd(m2, 256, 4), FC_ERR_CAPACITY);
    m2 = md;
    m2.merge = 0;
    EXPECT(mfwd(m2, 256, 1), FC_ERR_INVALID_ARG);
    m2 = md;
    m2.d_model = 1300;
    EXPECT(mfwd(m2, 256, 1), FC_ERR_SHAPE);
    m2 = md;
    m2.d_out = 3580;
    EXPECT(mfwd(m2, 256, 1), FC_ERR_SHAPE);
    m2 = md;
    m2.rms_eps = 0.f;
    EXPECT(mfwd(m2, 256, 1), FC_ERR_INVALID_ARG);
    m2 = md;
    m2.w2 = nullptr;
    EXPECT(mfwd(m2, 256, 1), FC_ERR_INVALID_ARG);
  }
  EXPECT(fc_profile_enable(nullptr, 1), FC_ERR_INVALID_ARG);
  EXPECT(fc_profile_only(nullptr, "k"), FC_ERR_INVALID_ARG);
  {
    double ms = 0;
    int64_t n = 0;
    EXPECT(fc_profile_read(nullptr, "k", &ms, &n, 0), FC_ERR_INVALID_ARG);
    EXPECT(fc_profile_only(ctx, "k_wgemm"), FC_OK);
    EXPECT(fc_profile_read(ctx, "k_wgemm", &ms, &n, 1), FC_OK);
    if (ms != 0 || n != 0) { std::printf("FAIL: records of an unused context\n"); ++g_fail; }
  }
  delete ctx;                                  // no device buffers to free

  std::printf("%s (%d failed expectations)\n", g_fail ? "FAILED" : "OK", g_fail);
  return g_fail ? 1 : 0;
}
