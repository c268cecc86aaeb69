// Slot-mapped token caches: K/V rows addressed through a per-item row map, so that a
// reused token (Sec. 4.1: it takes the cached results of its aligned source token,
// Eq. 4-2) shares its source's pool row instead of receiving a copy of it, in every
// layer at once (one map serves all layers of an item).
//
// State of one item (int32, in one caller buffer for B items, part after part):
//   map  [B][S]  pool row of every cache row; text rows and the rows after the frames
//                map to themselves, frame rows to pool rows in [T, T + W N)
//   ref  [B][S]  number of frame rows that map to each pool row
//   free [B][S]  stack of unreferenced frame pool rows (first `top` entries)
//   top  [B]
// At most W N frame rows are live, so the W N frame pool rows always suffice: a step
// releases the rows of the frame that leaves the window before it takes new ones.
#include <hip/hip_runtime.h>

#include "fc_internal.h"

namespace fc {
namespace {

constexpr int kSlotThreads = 1024;   // one thread per token of a frame (N <= 1024)

__global__ __launch_bounds__(256) void k_slot_init(int32_t *state, int B, int S, int T, int WN) {
  const int b = blockIdx.y;
  SlotState s = slot_state_at(state, B, S);
  for (int r = blockIdx.x * blockDim.x + threadIdx.x; r < S; r += gridDim.x * blockDim.x) {
    s.map[(long)b * S + r] = r;
    s.ref[(long)b * S + r] = (r >= T && r < T + WN) ? 1 : 0;
    s.free[(long)b * S + r] = 0;
  }
  if (blockIdx.x == 0 && threadIdx.x == 0) s.top[b] = 0;
}

// Block-wide exclusive prefix sum of a 0/1 flag in token order; returns the prefix and
// stores the total in *tot (all threads see it after the call).
__device__ int block_scan(int f, int *wsum, int *tot) {
  const int t = threadIdx.x, lane = t & 63, w = t >> 6;
  const unsigned long long m = __ballot(f);
  const int pre = __popcll(m & ((1ull << lane) - 1ull));
  if (lane == 0) wsum[w] = __popcll(m);
  __syncthreads();
  int base = 0, all = 0;
  for (int i = 0; i < (int)(blockDim.x >> 6); ++i) {
    if (i < w) base += wsum[i];
    all += wsum[i];
  }
  __syncthreads();
  *tot = all;
  return base + pre;
}

// One step of one item, after the window advanced (cur_row0: first row of the current
// frame's slot, prev_row0: of the previous frame's, equal for a one-frame window).
__global__ __launch_bounds__(kSlotThreads) void k_slot_remap(int32_t *state, int B, int S, int N,
                                                             int gw, int cur_row0, int prev_row0,
                                                             const int32_t *__restrict__ shift,
                                                             const uint8_t *__restrict__ reuse) {
  __shared__ int wsum[kSlotThreads / 64];
  const int b = blockIdx.x, tok = threadIdx.x;
  SlotState s = slot_state_at(state, B, S);
  int32_t *map = s.map + (long)b * S;
  int32_t *ref = s.ref + (long)b * S;
  int32_t *fre = s.free + (long)b * S;
  const bool live = tok < N;
  const int gh = N / gw;
  // 1. read everything the step replaces: the leaving frame's pool rows and, for
  //    reused tokens, their source rows (with one frame slot these are the same rows)
  // (pool rows outside [0, S) can only come from a state that k_slot_init never set up;
  // they are ignored rather than followed)
  int old = -1, src = -1;
  bool reused = false;
  if (live) {
    old = map[cur_row0 + tok];
    if (old < 0 || old >= S) old = -1;
    if (reuse[(long)b * N + tok]) {
      const int I = tok / gw, J = tok - I * gw;
      const int si = I + shift[2 * b], sj = J + shift[2 * b + 1];
      if (si >= 0 && si < gh && sj >= 0 && sj < gw) {
        src = map[prev_row0 + si * gw + sj];
        reused = src >= 0 && src < S;
      }
    }
  }
  __syncthreads();
  // 2. the reusers' references first, so that a row both left and reused survives
  if (reused) atomicAdd(&ref[src], 1);
  __syncthreads();
  bool freed = false;
  if (old >= 0) freed = atomicSub(&ref[old], 1) == 1;
  __syncthreads();
  // 3. push the freed rows (in token order), then pop one per recomputed token
  int nfree = 0;
  const int top0 = min(max(s.top[b], 0), S);
  const int fpos = block_scan(freed ? 1 : 0, wsum, &nfree);
  if (freed && top0 + fpos < S) fre[top0 + fpos] = old;
  __syncthreads();
  const int top1 = min(top0 + nfree, S);
  int nnew = 0;
  const bool fresh = live && !reused;
  const int npos = block_scan(fresh ? 1 : 0, wsum, &nnew);
  int row = src;
  if (fresh) {
    const int k = top1 - 1 - npos;
    row = (k >= 0 && k < S) ? fre[k] : -1;
    if (row < 0 || row >= S) row = cur_row0 + tok;   // never with a consistent state
    else ref[row] = 1;
  }
  if (live) map[cur_row0 + tok] = row;
  if (tok == 0) s.top[b] = max(top1 - nnew, 0);
}

}  // namespace

size_t slot_state_bytes(long B, long S) {
  if (B < 1 || S < 1 || (unsigned long)B * (unsigned long)S > (1UL << 40)) return 0;
  return (size_t)(3 * B * S + B) * sizeof(int32_t);
}

fc_status launch_slot_init(fc_ctx *ctx, const fc_kv_cache &kv, int B, hipStream_t st) {
  const int S = kv.text_tokens + kv.window * kv.frame_tokens + kv.trail_tokens;
  ProfScope ps(ctx, st, "fc_slot_init");
  hipLaunchKernelGGL(k_slot_init, dim3((unsigned)((S + 255) / 256), (unsigned)B), dim3(256), 0, st,
                     kv.slot_map, B, S, kv.text_tokens, kv.window * kv.frame_tokens);
  FC_LAUNCH_OK(st, "k_slot_init");
  return FC_OK;
}

fc_status launch_slot_remap(fc_ctx *ctx, const fc_kv_cache &kv, const int32_t *shift,
                            const uint8_t *reuse, int grid_w, int B, hipStream_t st) {
  const int N = kv.frame_tokens;
  const int S = kv.text_tokens + kv.window * N + kv.trail_tokens;
  if (N > kSlotThreads)
    return fail(FC_ERR_UNSUPPORTED, "slot map: N=%d tokens per frame > %d", N, kSlotThreads);
  const int cur_slot = (kv.head + kv.window - 1) % kv.window;
  const int prev_slot = kv.window > 1 ? (kv.head + kv.window - 2) % kv.window : cur_slot;
  ProfScope ps(ctx, st, "fc_slot_remap");
  hipLaunchKernelGGL(k_slot_remap, dim3((unsigned)B), dim3(kSlotThreads), 0, st, kv.slot_map, B, S,
                     N, grid_w, kv.text_tokens + cur_slot * N, kv.text_tokens + prev_slot * N,
                     shift, reuse);
  FC_LAUNCH_OK(st, "k_slot_remap");
  return FC_OK;
}

}  // namespace fc
