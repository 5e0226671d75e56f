// Greedy acceptance walk (temperature 0): accept the longest root path whose every node
// carries the target model's greedy token after its parent (Sec. 1: each round commits
// one prefix path; Limitations: greedy verification).
//
// One wavefront per request.  Each lane first evaluates "token[i] equals the target
// token after parent[i]" for its nodes; then the walk descends from the root, finding
// the unique matching child of the current node with one ballot per level (siblings
// carry distinct tokens, so at most one child matches).
#include "common.h"

namespace taps {

namespace {

// One request per wave; SLOTS = ceil(budget / 64) nodes per lane.
template <int SLOTS>
__global__ __launch_bounds__(kWave) void walk_kernel(const int32_t* __restrict__ parent,
                                                     const int32_t* __restrict__ token,
                                                     const int32_t* __restrict__ nn, int N,
                                                     int D, const int32_t* __restrict__ target,
                                                     int32_t* __restrict__ path,
                                                     int32_t* __restrict__ path_len,
                                                     int32_t* __restrict__ bonus) {
  __shared__ int32_t s_tgt[SLOTS * kWave];
  asm volatile("" ::"s"(parent), "s"(token), "s"(nn), "s"(N), "s"(D), "s"(target), "s"(path),
               "s"(path_len), "s"(bonus));
  const int b = blockIdx.x;
  const int lane = threadIdx.x;
  const int32_t* par = parent + (size_t)b * N;
  const int32_t* tok = token + (size_t)b * N;
  const int32_t* tgt = target + (size_t)b * N;

  // every node's parent, token and target token in one round of loads (clamped indices,
  // masked below); the node count is not needed to address them
  int p[SLOTS], tk[SLOTS], tg[SLOTS];
#pragma unroll
  for (int s = 0; s < SLOTS; ++s) {
    const int ic = min(s * kWave + lane, N - 1);
    p[s] = par[ic];
    tk[s] = tok[ic];
    tg[s] = tgt[ic];
  }
  const int n = min(max(nn[b], 1), N);
  // target tokens through LDS, so that each node can read its parent's
#pragma unroll
  for (int s = 0; s < SLOTS; ++s) s_tgt[s * kWave + lane] = tg[s];
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  // "token[i] equals the target token after parent[i]" for the request's nodes
  bool match[SLOTS];
#pragma unroll
  for (int s = 0; s < SLOTS; ++s) {
    const int i = s * kWave + lane;
    const bool valid = i >= 1 && i < n && p[s] >= 0 && p[s] < i;
    const int pt = s_tgt[valid ? p[s] : 0];
    match[s] = valid && tk[s] == pt;
    p[s] = valid ? p[s] : -1;
  }
  int cur = 0, len = 1;
  int32_t* out = path + (size_t)b * (D + 1);
  if (lane == 0) out[0] = 0;
  for (int step = 0; step < D; ++step) {
    int found = -1;
#pragma unroll
    for (int s = 0; s < SLOTS; ++s) {
      const uint64_t bal = __ballot(match[s] && p[s] == cur);
      if (found < 0 && bal) found = s * kWave + __ffsll((long long)bal) - 1;
    }
    if (found < 0) break;
    cur = found;
    if (lane == 0) out[len] = cur;
    ++len;
  }
  for (int j = len + lane; j <= D; j += kWave) out[j] = -1;
  if (lane == 0) {
    path_len[b] = len;
    bonus[b] = s_tgt[cur];
  }
}

}  // namespace

hipError_t launch_walk(const taps_tree& t, int batch, int budget, int block,
                       const int32_t* target, int32_t* path, int32_t* path_len, int32_t* bonus,
                       hipStream_t s) {
  if (batch <= 0) return hipSuccess;
  const dim3 grid((unsigned)batch), blk(kWave);
#define TAPS_WALK(SL)                                                                        \
  walk_kernel<SL><<<grid, blk, 0, s>>>(t.parent, t.token, t.n_nodes, budget, block, target, \
                                       path, path_len, bonus)
  static_assert(TAPS_MAX_BUDGET <= 8 * kWave, "at most eight node slots per lane");
  switch ((budget + kWave - 1) / kWave) {
    case 1: TAPS_WALK(1); break;
    case 2: TAPS_WALK(2); break;
    case 3:
    case 4: TAPS_WALK(4); break;
    default: TAPS_WALK(8); break;
  }
#undef TAPS_WALK
  return hipGetLastError();
}

}  // namespace taps
