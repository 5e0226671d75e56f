// Target-aware selection of one request per workgroup (Sec. 4.2-4.3, Eq. 1-3, Alg. 1).
//
// Phase A  merge the per-chunk top-K lists of each row into the row's top-K (one wave
//          per row): a threshold at the K-th largest chunk head keeps only the few
//          entries that can still be in the top-K; those are ranked exactly.
// Phase B  sibling-softmax edge probabilities c[i][r] (Eq. 1) in IEEE fp64 and the
//          utility denominators lambda1 + lambda2*d (Eq. 3).
// Phase C  greedy selection (Alg. 1) by one wave.  Because q_cond <= 1 and the
//          denominators do not decrease with depth, a child never beats its parent,
//          so the argmax of Alg. 1 always lies among the not-yet-selected children of
//          selected nodes.  Children of one node are offered in rank order (their
//          utilities do not increase with rank), so the candidates form one sorted list
//          per selected node; every pop takes the best list head.  Ties go to the
//          shallower node, then to the lexicographically smaller rank path.
// Phase D  write the tree.
//
// This file is compiled with -ffp-contract=off: every product and sum is rounded on
// its own, as in the definition both sides of the parity test implement.
#include "common.h"

namespace taps {

namespace {

constexpr int kThreads = 1024;
constexpr int kWaves = kThreads / kWave;
constexpr int kRowCap = TAPS_MAX_K * TAPS_MAX_K;  // entries >= the threshold, at most K*K

// ------------------------------------------------------------------ shared exponential
// Cody & Waite (1980) reduction t = k ln2 + r with ln2 = LN2_HI + LN2_LO (LN2_HI has 32
// significant bits, so k*LN2_HI is exact), then the degree-13 Taylor polynomial of
// exp(r) by Horner with coefficients 1/n! rounded to double, no fused multiply-add.
__host__ __device__ inline double spec_exp(double t) {
  const double INV_LN2 = 0x1.71547652b82fep+0;  // 1/ln2 rounded to nearest
  const double LN2_HI = 0x1.62e42ffp-1;         // ln2 rounded to 32 significant bits
  const double LN2_LO = -0x1.718432a1b0e26p-35; // ln2 - LN2_HI rounded to nearest
  const double C[14] = {
      0x1p+0,                 0x1p+0,                 0x1p-1,
      0x1.5555555555555p-3,   0x1.5555555555555p-5,   0x1.1111111111111p-7,
      0x1.6c16c16c16c17p-10,  0x1.a01a01a01a01ap-13,  0x1.a01a01a01a01ap-16,
      0x1.71de3a556c734p-19,  0x1.27e4fb7789f5cp-22,  0x1.ae64567f544e4p-26,
      0x1.1eed8eff8d898p-29,  0x1.6124613a86d09p-33};
  if (t != t || t < -708.0) return 0.0;
  if (t == 0.0) return 1.0;
  const double kf = rint(t * INV_LN2);
  const double r = (t - kf * LN2_HI) - kf * LN2_LO;
  double p = C[13];
  for (int n = 12; n >= 0; --n) p = p * r + C[n];
  return ldexp(p, (int)kf);
}

__device__ inline uint64_t shfl_u64(uint64_t v, int src) {
  uint32_t lo = __shfl((uint32_t)v, src), hi = __shfl((uint32_t)(v >> 32), src);
  return ((uint64_t)hi << 32) | lo;
}
__device__ inline uint64_t wave_max_u64(uint64_t v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) {
    uint32_t lo = __shfl_xor((uint32_t)v, m), hi = __shfl_xor((uint32_t)(v >> 32), m);
    uint64_t o = ((uint64_t)hi << 32) | lo;
    v = o > v ? o : v;
  }
  return v;
}
__device__ inline uint32_t wave_min_u32(uint32_t v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) {
    uint32_t o = __shfl_xor(v, m);
    v = o < v ? o : v;
  }
  return v;
}

// utility key: order-preserving bits of a non-negative double, shifted so 0 means "none"
__device__ inline uint64_t ukey(double u) { return (uint64_t)__double_as_longlong(u) + 1ull; }

__device__ inline float value_from_key(uint32_t vk) {
  if (vk == 0u) return __uint_as_float(0x7FC00000u);
  return __uint_as_float((vk & 0x80000000u) ? (vk & 0x7FFFFFFFu) : ~vk);
}

template <int SLOTS>
__global__ __launch_bounds__(kThreads) void select_kernel(
    int D, int K, int N, int kind, double lambda1, double lambda2, double tau, double beta,
    int chunks, const uint64_t* __restrict__ cand, int32_t* __restrict__ o_parent,
    int32_t* __restrict__ o_token, int32_t* __restrict__ o_depth, int32_t* __restrict__ o_rank,
    double* __restrict__ o_q, int32_t* __restrict__ o_n, int32_t* __restrict__ o_tidx,
    float* __restrict__ o_tval) {
  __shared__ uint64_t s_row[kWaves][kRowCap];
  __shared__ uint64_t s_top[TAPS_MAX_BLOCK][TAPS_MAX_K];
  __shared__ double s_e[TAPS_MAX_BLOCK][TAPS_MAX_K];
  __shared__ double s_c[TAPS_MAX_BLOCK][TAPS_MAX_K];
  __shared__ double s_den[TAPS_MAX_BLOCK + 1];
  // per selected node: candidate children keys and q, path digits, depth
  __shared__ uint64_t s_U[TAPS_MAX_BUDGET][TAPS_MAX_K];
  __shared__ double s_Q[TAPS_MAX_BUDGET][TAPS_MAX_K];
  __shared__ uint32_t s_path[TAPS_MAX_BUDGET][4];
  __shared__ int s_depth[TAPS_MAX_BUDGET], s_par[TAPS_MAX_BUDGET], s_rank[TAPS_MAX_BUDGET];
  __shared__ int s_n;

  const int b = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;

  // ---------------- Phase A: row merge
  for (int i = wave; i < D; i += kWaves) {
    const uint64_t* rc = cand + ((size_t)b * D + i) * chunks * K;
    // K-th largest chunk head (chunks <= 64, one per lane)
    const uint64_t head = lane < chunks ? rc[(size_t)lane * K] : 0ull;
    int beat = 0;
    for (int j = 0; j < chunks; ++j) beat += shfl_u64(head, j) > head ? 1 : 0;
    const int nheads = __popcll(__ballot(head != 0ull));
    uint64_t T;
    if (nheads >= K) {
      const uint64_t sel = __ballot(head != 0ull && beat == K - 1);
      T = shfl_u64(head, __ffsll((long long)sel) - 1);
    } else {
      T = 1ull;  // fewer non-empty chunks than K: every entry is a candidate
    }
    // gather entries >= T (each chunk list is sorted, at most K*K survive)
    int cnt = 0;
    for (int e = lane; e < chunks * K; e += kWave) cnt += rc[e] >= T ? 1 : 0;
    int incl = cnt;
    for (int off = 1; off < kWave; off <<= 1) {
      const int o = __shfl_up(incl, off);
      if (lane >= off) incl += o;
    }
    const int total = min(__shfl(incl, kWave - 1), kRowCap);
    int pos = incl - cnt;
    for (int e = lane; e < chunks * K; e += kWave) {
      const uint64_t v = rc[e];
      if (v >= T) {
        if (pos < kRowCap) s_row[wave][pos] = v;
        ++pos;
      }
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
    for (int c0 = 0; c0 < total; c0 += kWave) {
      const int me = c0 + lane;
      const uint64_t mine = me < total ? s_row[wave][me] : 0ull;
      int rank = 0;
      for (int j = 0; j < total; ++j) rank += s_row[wave][j] > mine ? 1 : 0;
      if (me < total && rank < K) s_top[i][rank] = mine;
    }
    for (int r = total + lane; r < K; r += kWave) s_top[i][r] = 0ull;
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
    if (lane < K) {
      const uint64_t k = s_top[i][lane];
      const size_t o = ((size_t)b * D + i) * K + lane;
      o_tidx[o] = k ? (int32_t)cand_index(k) : -1;
      if (o_tval) o_tval[o] = value_from_key((uint32_t)(k >> 32));
    }
  }
  __syncthreads();

  // ---------------- Phase B: Eq. 1 edge probabilities, Eq. 3 denominators
  if (tid < D * K) {
    const int i = tid / K, r = tid - (tid / K) * K;
    const uint64_t k = s_top[i][r];
    const double x = k ? (double)value_from_key((uint32_t)(k >> 32)) : (double)__uint_as_float(0x7FC00000u);
    double e;
    if (kind == TAPS_LOGITS) {
      const uint64_t k0 = s_top[i][0];
      const double x0 = k0 ? (double)value_from_key((uint32_t)(k0 >> 32)) : x;
      e = spec_exp(beta * (x - x0));
    } else {
      e = x > 0.0 ? x : 0.0;
    }
    s_e[i][r] = e;
  }
  if (tid <= D) s_den[tid] = lambda1 + lambda2 * (double)tid;
  __syncthreads();
  if (tid < D * K) {
    const int i = tid / K, r = tid - (tid / K) * K;
    double Z = 0.0;
    for (int j = 0; j < K; ++j) Z = Z + s_e[i][j];
    const bool ok = Z > 0.0 && Z <= 1.7976931348623157e308;
    s_c[i][r] = ok ? s_e[i][r] / Z : 0.0;
  }
  __syncthreads();

  // ---------------- Phase C: greedy selection (wave 0)
  if (wave == 0) {
    // root (node 0): its K children form list 0
    if (lane < K) {
      const double q = 1.0 * s_c[0][lane];
      s_Q[0][lane] = q;
      s_U[0][lane] = ukey(q / s_den[1]);
    }
    if (lane == 0) {
      s_depth[0] = 0; s_par[0] = -1; s_rank[0] = -1;
      s_path[0][0] = s_path[0][1] = s_path[0][2] = s_path[0][3] = 0u;
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
    uint64_t head[SLOTS];
    int nxt[SLOTS];
#pragma unroll
    for (int s = 0; s < SLOTS; ++s) { head[s] = 0ull; nxt[s] = 0; }
    if (lane == 0) head[0] = s_U[0][0];
    int m = 1;
    while (m < N) {
      // lane-local best list head
      uint64_t best = 0ull;
#pragma unroll
      for (int s = 0; s < SLOTS; ++s) best = head[s] > best ? head[s] : best;
      const uint64_t mx = wave_max_u64(best);
      if (mx == 0ull) break;
      const double umax = __longlong_as_double((long long)(mx - 1ull));
      if (!(umax > tau)) break;
      // entries holding the maximum; pick by (depth asc, rank path asc) on ties
      int ntie = 0, myslot = -1;
#pragma unroll
      for (int s = 0; s < SLOTS; ++s) {
        const bool t = head[s] == mx;
        ntie += __popcll(__ballot(t));
        if (t && myslot < 0) myslot = s;
      }
      int win;
      if (ntie == 1) {
        const uint64_t bal = __ballot(myslot >= 0);
        const int wl = __ffsll((long long)bal) - 1;
        const int ws = __shfl(myslot, wl);
        win = ws * kWave + wl;
      } else {
        // candidate child of entry j = node j's next rank: compare depth, then path words
        uint32_t key[SLOTS][5];
#pragma unroll
        for (int s = 0; s < SLOTS; ++s) {
          const int j = s * kWave + lane;
          if (head[s] == mx) {
            const int d = s_depth[j] + 1;
            key[s][0] = (uint32_t)d;
#pragma unroll
            for (int w = 0; w < 4; ++w) key[s][w + 1] = s_path[j][w];
            const int lvl = d - 1;  // digit position (0-based level)
            key[s][1 + lvl / 8] |= (uint32_t)nxt[s] << (28 - 4 * (lvl % 8));
          } else {
#pragma unroll
            for (int w = 0; w < 5; ++w) key[s][w] = 0xFFFFFFFFu;
          }
        }
        bool alive[SLOTS];
#pragma unroll
        for (int s = 0; s < SLOTS; ++s) alive[s] = head[s] == mx;
#pragma unroll
        for (int w = 0; w < 5; ++w) {
          uint32_t mn = 0xFFFFFFFFu;
#pragma unroll
          for (int s = 0; s < SLOTS; ++s) if (alive[s] && key[s][w] < mn) mn = key[s][w];
          mn = wave_min_u32(mn);
#pragma unroll
          for (int s = 0; s < SLOTS; ++s) alive[s] = alive[s] && key[s][w] == mn;
        }
        int ws = -1;
#pragma unroll
        for (int s = 0; s < SLOTS; ++s) if (alive[s] && ws < 0) ws = s;
        const uint64_t bal = __ballot(ws >= 0);
        const int wl = __ffsll((long long)bal) - 1;
        win = __shfl(ws, wl) * kWave + wl;
      }
      // emit node m = child (win, nxt[win]) and build its children list
      const int wlane = win % kWave, wslot = win / kWave;
      int r_w = 0;
#pragma unroll
      for (int s = 0; s < SLOTS; ++s) if (s == wslot) r_w = nxt[s];
      r_w = __shfl(r_w, wlane);
      const double qm = s_Q[win][r_w];
      const int dm = s_depth[win] + 1;
      if (lane == 0) {
        s_depth[m] = dm; s_par[m] = win; s_rank[m] = r_w;
#pragma unroll
        for (int w = 0; w < 4; ++w) s_path[m][w] = s_path[win][w];
        const int lvl = dm - 1;
        s_path[m][lvl / 8] |= (uint32_t)r_w << (28 - 4 * (lvl % 8));
      }
      if (lane < K) {
        if (dm < D) {
          const double q = qm * s_c[dm][lane];
          s_Q[m][lane] = q;
          s_U[m][lane] = ukey(q / s_den[dm + 1]);
        } else {
          s_Q[m][lane] = 0.0;
          s_U[m][lane] = 0ull;
        }
      }
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup");
      __builtin_amdgcn_wave_barrier();
      __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup");
      // advance the winner's list, open the new node's list
      const int mlane = m % kWave, mslot = m / kWave;
#pragma unroll
      for (int s = 0; s < SLOTS; ++s) {
        if (lane == wlane && s == wslot) {
          nxt[s] = r_w + 1;
          head[s] = nxt[s] < K ? s_U[win][nxt[s]] : 0ull;
        }
        if (lane == mlane && s == mslot) {
          nxt[s] = 0;
          head[s] = s_U[m][0];
        }
      }
      ++m;
    }
    if (lane == 0) s_n = m;
  }
  __syncthreads();

  // ---------------- Phase D: write the tree
  const int n = s_n;
  for (int j = tid; j < N; j += kThreads) {
    const size_t o = (size_t)b * N + j;
    if (j < n) {
      const int d = s_depth[j];
      o_parent[o] = s_par[j];
      o_depth[o] = d;
      o_rank[o] = s_rank[j];
      o_token[o] = j == 0 ? -1 : (int32_t)cand_index(s_top[d - 1][s_rank[j]]);
      o_q[o] = j == 0 ? 1.0 : s_Q[s_par[j]][s_rank[j]];
    } else {
      o_parent[o] = -1; o_depth[o] = -1; o_rank[o] = -1; o_token[o] = -1; o_q[o] = 0.0;
    }
  }
  if (tid == 0) o_n[b] = n;
}

}  // namespace

double spec_exp_host(double t) { return spec_exp(t); }

hipError_t launch_select(const void* /*marg*/, const taps_select_params& p, const TopkPlan& plan,
                         const uint64_t* cand, const taps_tree& out, hipStream_t s) {
  dim3 grid((unsigned)p.batch), block(kThreads);
  const int slots = (p.budget + kWave - 1) / kWave;
#define TAPS_SEL(SL)                                                                          \
  select_kernel<SL><<<grid, block, 0, s>>>(p.block, p.K, p.budget, p.kind, p.lambda1,         \
                                           p.lambda2, p.tau, p.beta, plan.chunks, cand,       \
                                           out.parent, out.token, out.depth, out.rank,        \
                                           out.q_reach, out.n_nodes, out.topk_idx, out.topk_val)
  switch (slots) {
    case 1: TAPS_SEL(1); break;
    case 2: TAPS_SEL(2); break;
    case 3: TAPS_SEL(3); break;
    default: TAPS_SEL(4); break;
  }
#undef TAPS_SEL
  return hipGetLastError();
}

}  // namespace taps
