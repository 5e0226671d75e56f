// Vocabulary-scan top-K (Sec. 4.1, Stage 1: the top-K tokens at each draft position).
//
// One workgroup scans one chunk of one marginal row and writes the chunk's K best
// 64-bit candidate keys (value key << 32 | ~index, larger is better, 0 = empty), sorted
// descending, to the workspace.  The selection kernel merges the chunks of a row.
//
// Per wave: every lane holds E values in registers (16-byte coalesced loads).  The
// K-th largest lane maximum T is found by a descent over its key bits with ballots; only
// values >= T can be in the wave's top-K, and there are few of them, so they are
// compacted into LDS and ranked exactly by counting.  A wave whose compacted set
// overflows falls back to K rounds of exact wave-wide argmax.  The four wave lists are
// merged by ranking again.
#include "common.h"

namespace taps {

namespace {

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / kWave;
constexpr int kWaveCap = 128;  // compacted candidates per wave before the fallback

__device__ inline uint64_t shfl_xor_u64(uint64_t v, int m) {
  uint32_t lo = __shfl_xor((uint32_t)v, m);
  uint32_t hi = __shfl_xor((uint32_t)(v >> 32), m);
  return ((uint64_t)hi << 32) | lo;
}

__device__ inline uint64_t wave_max_u64(uint64_t v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) {
    uint64_t o = shfl_xor_u64(v, m);
    v = o > v ? o : v;
  }
  return v;
}


// LDS exchange between the lanes of one wave (its LDS accesses execute in order)
__device__ inline void wave_fence_lds() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// inclusive prefix sum over the lanes of a wave (DPP row shifts, then row broadcasts)
__device__ inline int wave_inclusive_sum(int v) {
  v += __builtin_amdgcn_update_dpp(0, v, 0x111, 0xf, 0xf, false);  // row_shr:1
  v += __builtin_amdgcn_update_dpp(0, v, 0x112, 0xf, 0xf, false);  // row_shr:2
  v += __builtin_amdgcn_update_dpp(0, v, 0x114, 0xf, 0xf, false);  // row_shr:4
  v += __builtin_amdgcn_update_dpp(0, v, 0x118, 0xf, 0xf, false);  // row_shr:8
  v += __builtin_amdgcn_update_dpp(0, v, 0x142, 0xa, 0xf, false);  // row_bcast:15
  v += __builtin_amdgcn_update_dpp(0, v, 0x143, 0xc, 0xf, false);  // row_bcast:31
  return v;
}

template <int DT>
__device__ inline uint32_t elem_bits(const void* row, int64_t i) {
  if (DT == TAPS_BF16) return (uint32_t)((const uint16_t*)row)[i] << 16;
  return ((const uint32_t*)row)[i];
}

// Load element j of this thread: vector path covers 16-byte units u = t + 256*k.
template <int DT, int E>
__device__ inline void load_chunk(const void* row, bool aligned, int start, int end, int tid,
                                  uint32_t (&key)[E]) {
  constexpr int U = DT == TAPS_BF16 ? 8 : 4;  // elements per 16-byte unit
  if (aligned) {
#pragma unroll
    for (int k = 0; k < E / U; ++k) {
      const int e0 = start + (tid + kThreads * k) * U;
      if (e0 + U <= end) {
        const uint4 w = *(const uint4*)((const char*)row + (int64_t)e0 * (DT == TAPS_BF16 ? 2 : 4));
        const uint32_t ww[4] = {w.x, w.y, w.z, w.w};
        if (DT == TAPS_BF16) {
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            key[k * U + 2 * q] = value_key(ww[q] << 16);
            key[k * U + 2 * q + 1] = value_key(ww[q] & 0xFFFF0000u);
          }
        } else {
#pragma unroll
          for (int q = 0; q < 4; ++q) key[k * U + q] = value_key(ww[q]);
        }
      } else {
#pragma unroll
        for (int q = 0; q < U; ++q) {
          const int e = e0 + q;
          key[k * U + q] = e < end ? value_key(elem_bits<DT>(row, e)) : 0u;
        }
      }
    }
  } else {
#pragma unroll
    for (int j = 0; j < E; ++j) {
      const int e = start + tid + kThreads * j;
      key[j] = e < end ? value_key(elem_bits<DT>(row, e)) : 0u;
    }
  }
}

template <int DT, int E>
__device__ inline int elem_index(bool aligned, int start, int tid, int j) {
  constexpr int U = DT == TAPS_BF16 ? 8 : 4;
  return aligned ? start + (tid + kThreads * (j / U)) * U + (j % U) : start + tid + kThreads * j;
}

// Any chunk, any dtype: the wave's K best keys into s_wave_top[wave*K ...].
template <int DT, int E>
__device__ inline void generic_wave_topk(const void* rowp, bool aligned, int start, int end,
                                         int tid, int lane, int wave, int K, uint64_t* s_wc,
                                         uint64_t* s_wave_top) {
  uint32_t key[E];
  load_chunk<DT, E>(rowp, aligned, start, end, tid, key);
  // element keys are value keys; valid elements have an index < end.  Keys of missing
  // elements are 0 and are excluded by index below.
  uint32_t lmax = 0;
  bool any = false;
#pragma unroll
  for (int j = 0; j < E; ++j) {
    const bool ok = elem_index<DT, E>(aligned, start, tid, j) < end;
    any |= ok;
    lmax = (ok && key[j] >= lmax) ? key[j] : lmax;
  }
  // lanes without elements take no part in the threshold; a NaN-only lane takes part
  // with key 0
  const uint32_t lkey = any ? lmax : 0u;
  const bool has = any;
  // K-th largest lane maximum by bitwise descent (over value-key bits)
  uint32_t T = 0;
  const int nlanes = __popcll(__ballot(has));
  if (nlanes >= K) {
    constexpr int lowbit = DT == TAPS_BF16 ? 16 : 0;
    for (int bit = 31; bit >= lowbit; --bit) {
      const uint32_t c = T | (1u << bit);
      if (__popcll(__ballot(has && lkey >= c)) >= K) T = c;
    }
  }
  // compact all elements with key >= T (T = 0 keeps every valid element), in element
  // order, with one ballot per register slot
  int total = 0;
#pragma unroll
  for (int j = 0; j < E; ++j) {
    const int e = elem_index<DT, E>(aligned, start, tid, j);
    const bool c = key[j] >= T && e < end;
    const uint64_t m = __ballot(c);
    if (m) {
      const int pos = total + __builtin_amdgcn_mbcnt_hi((uint32_t)(m >> 32),
                                                        __builtin_amdgcn_mbcnt_lo((uint32_t)m, 0u));
      if (c && pos < kWaveCap) s_wc[pos] = cand_key(key[j], (uint32_t)e);
      total += __popcll(m);
    }
  }
  wave_fence_lds();

  if (total <= kWaveCap) {
    // exact rank of each compacted candidate within the wave
    for (int c0 = 0; c0 < total; c0 += kWave) {
      const int me = c0 + lane;
      const uint64_t mine = me < total ? s_wc[me] : 0ull;
      int rank = 0;
      for (int j0 = 0; j0 < total; j0 += 8) {
        uint64_t cv[8];
#pragma unroll
        for (int t = 0; t < 8; ++t) cv[t] = j0 + t < total ? s_wc[j0 + t] : 0ull;
#pragma unroll
        for (int t = 0; t < 8; ++t) rank += cv[t] > mine ? 1 : 0;
      }
      if (me < total && rank < K) s_wave_top[wave * K + rank] = mine;
    }
    for (int r = total + lane; r < K; r += kWave) s_wave_top[wave * K + r] = 0ull;
  } else {
    // fallback: K rounds of exact argmax over the wave's elements
    uint64_t prev = ~0ull;
    for (int r = 0; r < K; ++r) {
      uint64_t best = 0;
#pragma unroll
      for (int j = 0; j < E; ++j) {
        const int e = elem_index<DT, E>(aligned, start, tid, j);
        const uint64_t k = e < end ? cand_key(key[j], (uint32_t)e) : 0ull;
        best = (k < prev && k > best) ? k : best;
      }
      best = wave_max_u64(best);
      if (lane == 0) s_wave_top[wave * K + r] = best;
      prev = best;
    }
  }
}

// bf16 chunks whose length is a multiple of 8 and whose row is 16-byte aligned: the
// wave's candidates (every element that can be among its K best) into s_wc[0 .. *n_out).  Filtering uses float compares (NaN
// fails every compare, -0 equals +0, exactly like the integer keys); exact keys are built
// only for the few candidates.  Returns false (nothing written) when the wave has fewer
// than K non-NaN lanes or too many candidates; the generic path then takes the wave.
template <int E>
__device__ inline bool fast_wave_topk_bf16(const void* rowp, int start, int end, int tid,
                                           int K, uint64_t* s_wc, int* n_out) {
  static_assert(E % 8 == 0, "whole 16-byte units");
  // units past the chunk's end load an in-bounds unit and are replaced by NaN
  uint32_t w[E / 2];
#pragma unroll
  for (int k = 0; k < E / 8; ++k) {
    const int u = start + (tid + kThreads * k) * 8;
    const uint4 v = *(const uint4*)((const char*)rowp + (int64_t)min(u, end - 8) * 2);
    const bool in = u < end;
    w[4 * k] = in ? v.x : 0x7FC07FC0u;
    w[4 * k + 1] = in ? v.y : 0x7FC07FC0u;
    w[4 * k + 2] = in ? v.z : 0x7FC07FC0u;
    w[4 * k + 3] = in ? v.w : 0x7FC07FC0u;
  }
  float mx = -INFINITY;
#pragma unroll
  for (int j = 0; j < E / 2; ++j) {
    const float lo = __uint_as_float(w[j] << 16), hi = __uint_as_float(w[j] & 0xFFFF0000u);
    mx = fmaxf(mx, fmaxf(lo, hi));   // ignores NaN
  }
  // a lane takes part if it holds a non-NaN value; only a lane whose maximum is -inf
  // (all NaN, or -inf values) needs the element-wise test
  bool anynum = mx > -INFINITY;
  if (__ballot(!anynum)) {
#pragma unroll
    for (int j = 0; j < E / 2; ++j) {
      const float lo = __uint_as_float(w[j] << 16), hi = __uint_as_float(w[j] & 0xFFFF0000u);
      anynum |= lo == lo || hi == hi;
    }
  }
  if (__popcll(__ballot(anynum)) < K) return false;   // uniform
  // T: the largest 16-bit key with at least K lane maxima >= it, two bits per step
  const uint32_t lk = anynum ? (value_key(__float_as_uint(mx)) >> 16) : 0u;
  uint32_t T = 0;
#pragma unroll
  for (int b = 14; b >= 0; b -= 2) {
    const uint32_t c1 = T | (1u << b), c2 = T | (2u << b), c3 = T | (3u << b);
    const int n1 = __popcll(__ballot(lk >= c1));
    const int n2 = __popcll(__ballot(lk >= c2));
    const int n3 = __popcll(__ballot(lk >= c3));
    T = n3 >= K ? c3 : (n2 >= K ? c2 : (n1 >= K ? c1 : T));
  }
  const float tf = __uint_as_float((T & 0x8000u) ? ((T & 0x7FFFu) << 16) : (~(T << 16) & 0xFFFF0000u));
  // candidates (elements >= tf) of this lane as a bit mask over its elements, built with
  // vector operations only
  uint32_t mlo = 0u, mhi = 0u;
#pragma unroll
  for (int j = 0; j < E; ++j) {
    const uint32_t bits = (j & 1) ? (w[j >> 1] & 0xFFFF0000u) : (w[j >> 1] << 16);
    const uint32_t bit = __uint_as_float(bits) >= tf ? 1u : 0u;
    if (j < 32) mlo |= bit << (j & 31);
    else mhi |= bit << (j & 31);
  }
  const int c = __popc(mlo) + __popc(mhi);
  const int incl = wave_inclusive_sum(c);
  const int total = __builtin_amdgcn_readlane(incl, kWave - 1);
  if (total > kWaveCap) return false;   // uniform; rare (many ties)
  // compact: lane candidates go to positions incl - c ...; each round stores one
  // candidate per lane (the lane's lowest remaining element), reading its bits through a
  // select tree over the lane's words
  int pos = incl - c;
  while (__ballot((mlo | mhi) != 0u)) {
    if ((mlo | mhi) != 0u) {
      const int j = mlo ? __builtin_ctz(mlo) : 32 + __builtin_ctz(mhi);
      const int wi = j >> 1;
      uint32_t sel[E / 2];
#pragma unroll
      for (int i = 0; i < E / 2; ++i) sel[i] = w[i];
#pragma unroll
      for (int st = E / 4; st >= 1; st >>= 1) {
        const bool up = (wi & st) != 0;
#pragma unroll
        for (int i = 0; i < st; ++i) sel[i] = up ? sel[i + st] : sel[i];
      }
      const uint32_t bits = (j & 1) ? (sel[0] & 0xFFFF0000u) : (sel[0] << 16);
      const int e = start + (tid + kThreads * (j >> 3)) * 8 + (j & 7);
      s_wc[pos] = cand_key(value_key(bits), (uint32_t)e);
      ++pos;
      if (mlo) mlo &= mlo - 1u;
      else mhi &= mhi - 1u;
    }
  }
  *n_out = total;
  return true;
}

// The K best of a wave's `total` compacted candidates into s_top[0 .. K), in rank order
// (zero-padded): the rare path for workgroups with more than 64 candidates in all.
__device__ inline void rank_wave_candidates(const uint64_t* s_wc, int total, int K, int lane,
                                            uint64_t* s_top) {
  for (int c0 = 0; c0 < total; c0 += kWave) {
    const int me = c0 + lane;
    const uint64_t cx = s_wc[min(me, total - 1)];
    const uint64_t mine = me < total ? cx : 0ull;
    int rank = 0;
    for (int j0 = 0; j0 < total; j0 += 8) {
      uint64_t cv[8];
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        const uint64_t x = s_wc[min(j0 + t, total - 1)];
        cv[t] = j0 + t < total ? x : 0ull;
      }
#pragma unroll
      for (int t = 0; t < 8; ++t) rank += cv[t] > mine ? 1 : 0;
    }
    if (me < total && rank < K) s_top[rank] = mine;
  }
  for (int r = total + lane; r < K; r += kWave) s_top[r] = 0ull;
}

template <int DT, int E>
__global__ __launch_bounds__(kThreads) void topk_chunk_kernel(const void* __restrict__ marg,
                                                              int vocab, int K, int chunk_len,
                                                              int chunks,
                                                              uint64_t* __restrict__ cand) {
  __shared__ uint64_t s_cand[kWaves][kWaveCap];          // fast path: unranked candidates
  __shared__ uint64_t s_top[kWaves * TAPS_MAX_K];        // ranked lists: wave w's at w*K
  __shared__ int s_cnt[kWaves];                          // candidates of a fast-path wave, -1
                                                         // for a ranked list in s_top
  __shared__ uint64_t s_all[kWave];                      // the workgroup's candidates, one per
                                                         // lane of wave 0

  const int row = blockIdx.x / chunks;
  const int chunk = blockIdx.x - row * chunks;
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
  const int start = chunk * chunk_len;
  const int end = min(vocab, start + chunk_len);
  const size_t es = DT == TAPS_BF16 ? 2 : 4;
  const void* rowp = (const char*)marg + (size_t)row * vocab * es;
  const bool aligned = (((uintptr_t)rowp) & 15) == 0;

  int n = -1;
  if (DT == TAPS_BF16 && aligned && ((end - start) & 7) == 0 && end - start >= 8) {
    if (!fast_wave_topk_bf16<E>(rowp, start, end, tid, K, s_cand[wave], &n)) n = -1;
  }
  if (n < 0) generic_wave_topk<DT, E>(rowp, aligned, start, end, tid, lane, wave, K, s_cand[wave], s_top);
  if (lane == 0) s_cnt[wave] = n;
  __syncthreads();
  // list sizes: an unranked candidate list, or a ranked list of K in s_top
  int cnt[kWaves], tot = 0;
  bool all_ranked = false;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) {
    const int c = s_cnt[w];
    cnt[w] = c < 0 ? K : c;
    tot += cnt[w];
  }
  if (tot > kWave) {   // uniform, rare: every wave first cuts its candidates to its K best
    if (n >= 0) rank_wave_candidates(s_cand[wave], n, K, lane, s_top + wave * K);
    __syncthreads();
    all_ranked = true;
    tot = kWaves * K;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) cnt[w] = K;
  }
  if (wave != 0) return;
  // wave 0 ranks the (at most 64) entries of the four lists, one per lane
  int w = 0, off = 0;
#pragma unroll
  for (int v = 0; v < kWaves - 1; ++v)
    if (lane >= off + cnt[w]) { off += cnt[w]; ++w; }
  const bool in = lane < tot;
  const int wl = in ? w : 0, il = in ? lane - off : 0;
  const bool from_top = all_ranked || s_cnt[wl] < 0;
  const uint64_t cx = from_top ? s_top[wl * K + min(il, K - 1)] : s_cand[wl][il];
  const uint64_t mine = in ? cx : 0ull;
  // rank = candidates that beat this one, read back from LDS eight at a time (every lane
  // reads the same address; entries past tot are 0 and beat nothing)
  s_all[lane] = mine;
  wave_fence_lds();
  int rank = 0;
  for (int t0 = 0; t0 < tot; t0 += 8) {
    uint64_t v[8];
#pragma unroll
    for (int t = 0; t < 8; ++t) v[t] = s_all[t0 + t];
#pragma unroll
    for (int t = 0; t < 8; ++t) rank += v[t] > mine ? 1 : 0;
  }
  uint64_t* outp = cand + ((size_t)row * chunks + chunk) * K;
  if (in && mine != 0ull && rank < K) outp[rank] = mine;
  // ranks held by empty entries: write 0 (a chunk with fewer than K elements)
  const int nonempty = __popcll(__ballot(in && mine != 0ull));
  if (lane >= nonempty && lane < K) outp[lane] = 0ull;
}

template <int DT>
hipError_t launch_dt(const void* marg, int rows, int vocab, int K, const TopkPlan& p,
                     uint64_t* cand, hipStream_t s) {
  dim3 grid((unsigned)(rows * p.chunks)), block(kThreads);
  switch (p.per_thread) {
    case 8: topk_chunk_kernel<DT, 8><<<grid, block, 0, s>>>(marg, vocab, K, p.chunk_len, p.chunks, cand); break;
    case 16: topk_chunk_kernel<DT, 16><<<grid, block, 0, s>>>(marg, vocab, K, p.chunk_len, p.chunks, cand); break;
    case 32: topk_chunk_kernel<DT, 32><<<grid, block, 0, s>>>(marg, vocab, K, p.chunk_len, p.chunks, cand); break;
    default: topk_chunk_kernel<DT, 64><<<grid, block, 0, s>>>(marg, vocab, K, p.chunk_len, p.chunks, cand); break;
  }
  return hipGetLastError();
}

}  // namespace

TopkPlan plan_topk(int vocab, int rows, int /*dtype*/) {
  // aim for ~512 workgroups; chunks of 2048..16384 elements (8..64 per thread)
  const int target_chunks = rows >= 512 ? 1 : (512 + rows - 1) / rows;
  int len = 2048;
  while (len < 16384 &&
         ((int64_t)len * target_chunks < vocab || (vocab + len - 1) / len > 64))
    len *= 2;
  TopkPlan p;
  p.chunk_len = len;
  p.chunks = (vocab + len - 1) / len;
  p.per_thread = len / kThreads;
  return p;
}

hipError_t launch_topk_chunks(const void* marg, int dtype, int rows, int vocab, int K,
                              const TopkPlan& plan, uint64_t* cand, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  return dtype == TAPS_BF16 ? launch_dt<TAPS_BF16>(marg, rows, vocab, K, plan, cand, s)
                            : launch_dt<TAPS_FP32>(marg, rows, vocab, K, plan, cand, s);
}

}  // namespace taps
