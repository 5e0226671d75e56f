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

constexpr int kSlots = TAPS_MAX_BUDGET / kWave;

__global__ __launch_bounds__(kWave) void walk_kernel(const int32_t* __restrict__ parent,
                                                     const int32_t* __restrict__ token,
                                                     const int32_t* __restrict__ nn, int N,
                                                     int D, const int32_t* __restrict__ target,
                                                     int32_t* __restrict__ path,
                                                     int32_t* __restrict__ path_len,
                                                     int32_t* __restrict__ bonus) {
  const int b = blockIdx.x;
  const int lane = threadIdx.x;
  const int n = min(max(nn[b], 1), N);
  const int32_t* par = parent + (size_t)b * N;
  const int32_t* tok = token + (size_t)b * N;
  const int32_t* tgt = target + (size_t)b * N;

  int p[kSlots];
  bool match[kSlots];
#pragma unroll
  for (int s = 0; s < kSlots; ++s) {
    const int i = s * kWave + lane;
    p[s] = -1;
    match[s] = false;
    if (i >= 1 && i < n) {
      const int pi = par[i];
      if (pi >= 0 && pi < i) {
        p[s] = pi;
        match[s] = tok[i] == tgt[pi];
      }
    }
  }
  int cur = 0, len = 1;
  int32_t* out = path + (size_t)b * (D + 1);
  if (lane == 0) out[0] = 0;
  for (int step = 0; step < D; ++step) {
    int found = -1;
#pragma unroll
    for (int s = 0; s < kSlots; ++s) {
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
    bonus[b] = tgt[cur];
  }
}

}  // namespace

hipError_t launch_walk(const taps_tree& t, int batch, int budget, int block,
                       const int32_t* target, int32_t* path, int32_t* path_len, int32_t* bonus,
                       hipStream_t s) {
  if (batch <= 0) return hipSuccess;
  walk_kernel<<<dim3((unsigned)batch), dim3(kWave), 0, s>>>(t.parent, t.token, t.n_nodes, budget,
                                                          block, target, path, path_len, bonus);
  return hipGetLastError();
}

}  // namespace taps
