// Target-aware selection of one request per workgroup (Sec. 4.2-4.3, Eq. 1-3, Alg. 1).
//
// Phase A  merge the per-chunk top-K lists of each row into the row's top-K (one wave
//          per row): a threshold at the K-th largest chunk head keeps only the few
//          entries that can still be in the top-K (more than 64 of them are first cut
//          to the K largest by a descent over the key bits); those are ranked exactly.
//          The same wave then computes the row's sibling-softmax edge probabilities
//          c[i][r] (Eq. 1) in IEEE fp64.  The utility denominators lambda1 + lambda2*d
//          (Eq. 3) are set alongside.
// Phase C  the selected set of Alg. 1.  Because q_cond <= 1 and the denominators do not
//          decrease with depth, a child never beats its parent (ties go to the shallower
//          node), so Alg. 1 adds exactly one node per iteration and its result is the
//          first N-1 nodes of the trie in the order "utility descending, then depth
//          ascending, then rank path ascending" among those with utility > tau.
//          The trie is expanded one depth at a time, all candidates of a depth in
//          parallel.  A histogram of utilities over fixed bins (exponent and 3 mantissa
//          bits) gives a bin b* such that at least N-1 expanded nodes lie in bins >= b*;
//          any node below b* is beaten by N-1 others and so are its descendants, so it is
//          pruned.  At the end only the members of bin b* need an exact ranking.
//          Nodes are stored depth by depth, each depth in rank-path order, so the stored
//          index breaks ties between equal utilities exactly like the rank path does.
//          If the expansion outgrows its LDS capacity, a sequential best-first loop
//          computes the same set.
// Phase D  write the tree breadth first (depth, then rank path).
//
// This file is compiled with -ffp-contract=off: every product and sum is rounded on
// its own, as in the definition both sides of the parity test implement.
#include "common.h"

namespace taps {

namespace {

constexpr int kThreadsA = 1024;                   // Phase A: one wave per marginal row
constexpr int kWavesA = kThreadsA / kWave;
constexpr int kThreads = 256;                     // Phases B-D: four waves
constexpr int kWaves = kThreads / kWave;
constexpr int kRowCap = TAPS_MAX_K * TAPS_MAX_K;  // entries >= the threshold, at most K*K
constexpr int kCap = 3072;                        // expanded nodes held in LDS
constexpr int kBins = 1024;
constexpr int kCoarse = kBins / 16;
constexpr int kBinBase = (1023 - 110) * 8;        // bin 0 holds u < 2^-110

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

// ------------------------------------------------------------------ shared logarithm
// log x for finite x > 0: x = m 2^e, m in [sqrt(1/2), sqrt(2)); s = (m-1)/(m+1);
// log m = 2 s (1 + s^2/3 + ... + s^26/27) by Horner in s^2 (coefficients 1/(2k+1) rounded to
// double); result = e LN2_HI + (e LN2_LO + log m).  No fused multiply-add.
__host__ __device__ inline double spec_log(double x) {
  const double LN2_HI = 0x1.62e42ffp-1;
  const double LN2_LO = -0x1.718432a1b0e26p-35;
  const double SQRT_HALF = 0x1.6a09e667f3bcdp-1;
  int e;
  double m = frexp(x, &e);
  if (m < SQRT_HALF) {
    m = m * 2.0;
    e = e - 1;
  }
  const double s = (m - 1.0) / (m + 1.0);
  const double z = s * s;
  double p = 1.0 / 27.0;
  const double C[13] = {1.0, 1.0 / 3.0, 1.0 / 5.0, 1.0 / 7.0, 1.0 / 9.0, 1.0 / 11.0, 1.0 / 13.0,
                        1.0 / 15.0, 1.0 / 17.0, 1.0 / 19.0, 1.0 / 21.0, 1.0 / 23.0, 1.0 / 25.0};
  for (int k = 12; k >= 0; --k) p = p * z + C[k];
  const double logm = 2.0 * (s * p);
  const double ef = (double)e;
  return ef * LN2_HI + (ef * LN2_LO + logm);
}

template <int V>
struct IntC {
  static constexpr int value = V;
};

// ------------------------------------------------------------------ wave helpers
__device__ inline int lanes_below(uint64_t mask) {
  return __builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32),
                                   __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
}

// LDS exchange between the lanes of one wave: a wave's LDS accesses execute in order,
// so wavefront-scope ordering suffices (no wait for outstanding global loads)
__device__ inline void wave_fence() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// exclusive prefix of a small non-negative count (< 2^bits) over the lanes of a wave
template <int BITS>
__device__ inline int wave_prefix_small(int v, int& total) {
  int pre = 0, tot = 0;
#pragma unroll
  for (int b = 0; b < BITS; ++b) {
    const uint64_t m = __ballot((v >> b) & 1);
    pre += lanes_below(m) << b;
    tot += __popcll(m) << b;
  }
  total = tot;
  return pre;
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

// bitwise OR / AND over the lanes of a wave (DPP row shifts, then row broadcasts; lanes
// without a source keep the identity), read from the last lane
__device__ inline uint32_t wave_or_u32(uint32_t v) {
  v |= (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x111, 0xf, 0xf, false);
  v |= (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x112, 0xf, 0xf, false);
  v |= (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x114, 0xf, 0xf, false);
  v |= (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x118, 0xf, 0xf, false);
  v |= (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x142, 0xa, 0xf, false);
  v |= (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, 0x143, 0xc, 0xf, false);
  return (uint32_t)__builtin_amdgcn_readlane((int)v, kWave - 1);
}
__device__ inline uint32_t wave_and_u32(uint32_t v) {
  v &= (uint32_t)__builtin_amdgcn_update_dpp(-1, (int)v, 0x111, 0xf, 0xf, false);
  v &= (uint32_t)__builtin_amdgcn_update_dpp(-1, (int)v, 0x112, 0xf, 0xf, false);
  v &= (uint32_t)__builtin_amdgcn_update_dpp(-1, (int)v, 0x114, 0xf, 0xf, false);
  v &= (uint32_t)__builtin_amdgcn_update_dpp(-1, (int)v, 0x118, 0xf, 0xf, false);
  v &= (uint32_t)__builtin_amdgcn_update_dpp(-1, (int)v, 0x142, 0xa, 0xf, false);
  v &= (uint32_t)__builtin_amdgcn_update_dpp(-1, (int)v, 0x143, 0xc, 0xf, false);
  return (uint32_t)__builtin_amdgcn_readlane((int)v, kWave - 1);
}

// sum of a 64-bit integer over the lanes of a wave (exact), in every lane
__device__ inline int64_t wave_sum_i64(int64_t v) {
#pragma unroll
  for (int m = kWave / 2; m >= 1; m >>= 1) {
    const uint32_t lo = __shfl_xor((uint32_t)v, m), hi = __shfl_xor((uint32_t)((uint64_t)v >> 32), m);
    v += (int64_t)(((uint64_t)hi << 32) | lo);
  }
  return v;
}

// sum of a 64-bit integer over each 32-lane half of a wave (exact), in every lane of it
__device__ inline int64_t half_sum_i64(int64_t v) {
#pragma unroll
  for (int m = 16; m >= 1; m >>= 1) {
    const uint32_t lo = __shfl_xor((uint32_t)v, m), hi = __shfl_xor((uint32_t)((uint64_t)v >> 32), m);
    v += (int64_t)(((uint64_t)hi << 32) | lo);
  }
  return v;
}

// inclusive prefix sum within each row of 16 lanes
__device__ inline int row_inclusive_sum(int v) {
  v += __builtin_amdgcn_update_dpp(0, v, 0x111, 0xf, 0xf, false);  // row_shr:1
  v += __builtin_amdgcn_update_dpp(0, v, 0x112, 0xf, 0xf, false);  // row_shr:2
  v += __builtin_amdgcn_update_dpp(0, v, 0x114, 0xf, 0xf, false);  // row_shr:4
  v += __builtin_amdgcn_update_dpp(0, v, 0x118, 0xf, 0xf, false);  // row_shr:8
  return v;
}

// Exclusive prefix sum over the workgroup (every thread calls it, in uniform control
// flow).  The wave totals pass through one of two LDS slots, alternating per call: a slot
// is written again only two calls later, after every wave has passed the barrier of the
// call in between, so one barrier per call suffices.
__device__ inline int block_prefix(int v, int (*s_w)[kWaves], int& parity, int& total) {
  const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
  const int incl = wave_inclusive_sum(v);
  if (lane == kWave - 1) s_w[parity][wave] = incl;
  __syncthreads();
  int base = 0, tot = 0;
#pragma unroll
  for (int w = 0; w < kWaves; ++w) {
    const int x = s_w[parity][w];
    base += w < wave ? x : 0;
    tot += x;
  }
  parity ^= 1;
  total = tot;
  return base + incl - v;
}

// utility key: order-preserving bits of a non-negative double
__device__ inline uint64_t ubits(double u) { return (uint64_t)__double_as_longlong(u); }
__device__ inline int ubin(double u) {
  const int b = (int)(ubits(u) >> 49) - kBinBase;
  return b < 0 ? 0 : (b >= kBins ? kBins - 1 : b);
}

__device__ inline float value_from_key(uint32_t vk) {
  if (vk == 0u) return __uint_as_float(0x7FC00000u);
  return __uint_as_float((vk & 0x80000000u) ? (vk & 0x7FFFFFFFu) : ~vk);
}

// the value of lane l (wave-uniform l) in every lane
__device__ inline uint64_t read_lane_u64(uint64_t v, int l) {
  return ((uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)(v >> 32), l) << 32) |
         (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, l);
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

// ------------------------------------------------------------------ shared memory layout
struct PhaseA {
  uint64_t rowc[kWavesA][kRowCap];
  uint64_t heads[kWavesA][kWave + 2];   // two rows per wave: 33 entries per half
};
struct Level {                 // expanded trie nodes, stored depth by depth
  double q[kCap];
  uint64_t u[kCap];            // utility bits
  int meta[kCap];              // parent index << 16 | depth << 8 | rank
  union {
    int newidx[kCap];          // output position of each kept node
    uint64_t mkey[kCap];       // utility bits of the boundary bin's members, stored order
  };
  int hist[kBins];             // nodes per utility bin
  int chist[kCoarse];          // nodes per group of 16 bins
};
struct Seq {                   // sequential fallback, per selected node (selection order)
  double q[TAPS_MAX_BUDGET];                 // q_reach
  uint32_t path[TAPS_MAX_BUDGET][4];         // rank path, 4 bits per level from the root
  int depth[TAPS_MAX_BUDGET], par[TAPS_MAX_BUDGET], rank[TAPS_MAX_BUDGET];
  int order[TAPS_MAX_BUDGET];                // breadth-first position
  uint8_t ord[TAPS_MAX_BUDGET][TAPS_MAX_K];  // child ranks by (utility desc, rank asc)
};
union Scratch {
  PhaseA a;
  Level l;
  Seq s;
};
static_assert(kBins * 32 >= kCap, "one bit per boundary-bin member fits the histogram");

struct Shared {
  uint64_t top[TAPS_MAX_BLOCK][TAPS_MAX_K];
  double e[TAPS_MAX_BLOCK][TAPS_MAX_K];
  double c[TAPS_MAX_BLOCK][TAPS_MAX_K];
  double den[TAPS_MAX_BLOCK + 1];
  double lz[TAPS_MAX_BLOCK], ent[TAPS_MAX_BLOCK];   // learned scorer: LOG(Z), entropy
  int wsum[2][kWaves];
  int n;
  Scratch x;
};

// The pruning bin b*: the highest bin j such that at least N-1 expanded nodes lie in
// bins >= j (0 if there is none).  Every wave computes it from the two histograms: the
// coarse one picks the group of 16 bins, the fine one the bin within it.
__device__ inline int find_bstar(const Level& L, int N) {
  const int lane = threadIdx.x & (kWave - 1);
  static_assert(kCoarse == kWave, "one coarse bin per lane");
  const int incl = wave_inclusive_sum(L.chist[kCoarse - 1 - lane]);  // bins >= 16 (63 - lane)
  const uint64_t ok = __ballot(incl >= N - 1);
  if (ok == 0ull) return 0;
  const int l0 = __ffsll((long long)ok) - 1;
  const int C = kCoarse - 1 - l0;
  const int above = l0 > 0 ? __builtin_amdgcn_readlane(incl, l0 - 1) : 0;
  const int f = row_inclusive_sum(lane < 16 ? L.hist[C * 16 + 15 - lane] : 0);
  const uint64_t ok2 = __ballot(lane < 16 && above + f >= N - 1);
  return C * 16 + 15 - (__ffsll((long long)ok2) - 1);
}

// Weights of the learned-scorer hook (device fp32 arrays) and its sizes
struct ScorerArgs {
  const float* emb;          // [vocab][d]
  const float* W1;           // [h][2d + 3]
  const float* b1;           // [h]
  const float* w2;           // [h]
  float b2;
  const int32_t* root_token; // [batch]
  int d, h, vocab;
};

// Working set of the learned scorer in the scratch area: float counts of the weight block
// (W1, b1, w2) and of the embedding block (row stride ES), then four doubles per hidden unit
// (its three edge-feature weights and its w2), the parent slots np and all slots S of the
// hidden-unit parts, and the units KC per chunk (below 1: does not fit)
struct LearnedLayout {
  int wsz, ES, esz, np, S, KC;
};
__host__ __device__ inline LearnedLayout learned_layout(int D, int K, int d, int h) {
  LearnedLayout l;
  l.wsz = (h * (2 * d + 3) + 2 * h + 1) & ~1;
  l.ES = d | 1;
  l.esz = ((D * K + 1) * l.ES + 1) & ~1;
  l.np = 1 + (D - 1) * K;
  l.S = l.np + D * K;
  const long long left = (long long)sizeof(Scratch) - 4ll * (l.wsz + l.esz) - 32ll * h;
  const long long kc = left > 0 ? left / (8ll * l.S) : 0;
  l.KC = (int)(kc < h ? kc : h);
  return l;
}

// q_cond of the rank-r child of a depth-d node of rank pr (the root: pr = 0): the scorer's
// table c3[d][pr][r] for the learned scorer, else c[d][r]
__device__ inline double qcond(const Shared& sh, const double* c3, int K, int d, int pr, int r) {
  return c3 ? c3[(d * K + pr) * K + r] : sh.c[d][r];
}

// ------------------------------------------------------------------ Phase C fallback
// Sequential best-first selection (one wave) for expansions larger than kCap; emits S
// through sh.x.s in breadth-first order and returns n.  The frontier holds, for every
// selected node, its best child not yet selected: the children of a node are visited in
// the order (utility descending, rank ascending), which is the order Alg. 1's argmax and
// its tie-break give siblings.  With the sibling and marginal scorers that order is the
// rank order; the learned scorer's table need not fall with rank.  Lane l owns the nodes
// l, l + 64, ... (slot s: node s * 64 + l); head[s] holds the utility bits + 1 of that
// node's next child (0: none left), nxt[s] its position in the node's child order.
template <int SLOTS>
__device__ __attribute__((always_inline)) inline int select_sequential(Shared& sh, const double* c3,
                                                                     int D, int K, int N,
                                                                     double tau) {
  Seq& S = sh.x.s;
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
  if (wave == 0) {
    // utility key (bits + 1; 0: none) of the rank-r child of node j, whose rank is pr and
    // depth d (d < D)
    auto child_key = [&](int j, int d, int pr, int r) -> uint64_t {
      const double q = S.q[j] * qcond(sh, c3, K, d, pr, r);
      return ubits(q / sh.den[d + 1]) + 1ull;
    };
    // order the K children of node j (lanes < K, one child each) into S.ord[j]; returns, in
    // every lane, the key of the first child in that order
    auto order_children = [&](int j, int d, int pr) -> uint64_t {
      const uint64_t mine = lane < K && d < D ? child_key(j, d, pr, lane) : 0ull;
      int pos = 0;
      for (int r = 0; r < K; ++r) {
        const uint64_t o = read_lane_u64(mine, r);
        pos += (o > mine || (o == mine && r < lane)) ? 1 : 0;
      }
      if (lane < K) S.ord[j][pos] = (uint8_t)lane;
      const uint64_t first = __ballot(lane < K && pos == 0);
      return read_lane_u64(mine, __ffsll((long long)first) - 1);
    };
    if (lane == 0) {
      S.q[0] = 1.0;
      S.depth[0] = 0; S.par[0] = -1; S.rank[0] = -1;
      S.path[0][0] = S.path[0][1] = S.path[0][2] = S.path[0][3] = 0u;
    }
    wave_fence();
    uint64_t head[SLOTS];
    int nxt[SLOTS];
#pragma unroll
    for (int s = 0; s < SLOTS; ++s) { head[s] = 0ull; nxt[s] = 0; }
    {
      const uint64_t h0 = order_children(0, 0, 0);
      if (lane == 0) head[0] = h0;
    }
    wave_fence();
    int m = 1;
    while (m < N) {
      uint64_t best = 0ull;
#pragma unroll
      for (int s = 0; s < SLOTS; ++s) best = head[s] > best ? head[s] : best;
      const uint64_t mx = wave_max_u64(best);
      if (mx == 0ull) break;
      const double umax = __longlong_as_double((long long)(mx - 1ull));
      if (!(umax > tau)) break;
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
        win = __shfl(myslot, wl) * kWave + wl;
      } else {
        // equal utilities: the shallower child, then the smaller rank path
        uint32_t key[SLOTS][5];
        bool alive[SLOTS];
#pragma unroll
        for (int s = 0; s < SLOTS; ++s) {
          const int j = s * kWave + lane;
          alive[s] = head[s] == mx;
          if (alive[s]) {
            const int d = S.depth[j] + 1;
            key[s][0] = (uint32_t)d;
#pragma unroll
            for (int w = 0; w < 4; ++w) key[s][w + 1] = S.path[j][w];
            const int lvl = d - 1;
            key[s][1 + lvl / 8] |= (uint32_t)S.ord[j][nxt[s]] << (28 - 4 * (lvl % 8));
          } else {
#pragma unroll
            for (int w = 0; w < 5; ++w) key[s][w] = 0xFFFFFFFFu;
          }
        }
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
      const int wlane = win % kWave, wslot = win / kWave;
      int pos_w = 0;
#pragma unroll
      for (int s = 0; s < SLOTS; ++s) if (s == wslot) pos_w = nxt[s];
      pos_w = __shfl(pos_w, wlane);
      const int r_w = S.ord[win][pos_w];
      const int dw = S.depth[win];
      const int dm = dw + 1;
      if (lane == 0) {
        S.q[m] = S.q[win] * qcond(sh, c3, K, dw, dw == 0 ? 0 : S.rank[win], r_w);
        S.depth[m] = dm; S.par[m] = win; S.rank[m] = r_w;
#pragma unroll
        for (int w = 0; w < 4; ++w) S.path[m][w] = S.path[win][w];
        const int lvl = dm - 1;
        S.path[m][lvl / 8] |= (uint32_t)r_w << (28 - 4 * (lvl % 8));
      }
      wave_fence();
      const uint64_t hm = order_children(m, dm, r_w);   // 0 when dm == D
      // the winner's next child in its order
      uint64_t hw = 0ull;
      if (lane == wlane && pos_w + 1 < K)
        hw = child_key(win, dw, dw == 0 ? 0 : S.rank[win], S.ord[win][pos_w + 1]);
      const int mlane = m % kWave, mslot = m / kWave;
#pragma unroll
      for (int s = 0; s < SLOTS; ++s) {
        if (lane == wlane && s == wslot) {
          nxt[s] = pos_w + 1;
          head[s] = hw;
        }
        if (lane == mlane && s == mslot) {
          nxt[s] = 0;
          head[s] = hm;
        }
      }
      wave_fence();
      ++m;
    }
    if (lane == 0) sh.n = m;
  }
  __syncthreads();
  const int n = sh.n;
  // breadth-first position of every selected node: (depth, path) ascending
  for (int i = tid; i < n; i += kThreads) {
    int pos = 0;
    for (int j = 0; j < n; ++j) {
      bool less = S.depth[j] < S.depth[i];
      if (S.depth[j] == S.depth[i]) {
        int w = 0;
        while (w < 3 && S.path[j][w] == S.path[i][w]) ++w;
        less = S.path[j][w] < S.path[i][w];
      }
      pos += less ? 1 : 0;
    }
    S.order[i] = pos;
  }
  __syncthreads();
  return n;
}

// LEARNED: the learned scorer's instance (its q_cond table and Phase B2); the other
// scorers run an instance without that code, so their kernel stays smaller.
template <int SLOTS, bool LEARNED>
__global__ __launch_bounds__(kThreadsA) void select_kernel(
    int D, int K, int N, int kind, double lambda1, double lambda2, double tau, double beta,
    int chunks, int marginal, const uint64_t* __restrict__ cand,
    const int64_t* __restrict__ zpart, const int64_t* __restrict__ spart, ScorerArgs mlp,
    int32_t* __restrict__ o_parent,
    int32_t* __restrict__ o_token, int32_t* __restrict__ o_depth, int32_t* __restrict__ o_rank,
    double* __restrict__ o_q, int32_t* __restrict__ o_n, int32_t* __restrict__ o_tidx,
    float* __restrict__ o_tval) {
  __shared__ Shared sh;
  const int b = blockIdx.x;
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
  const bool learned = LEARNED && spart != nullptr;   // the entropy partials come with it

  // ---------------- Phase A: row merge (one wave per row)
  // Loads below take clamped (in-bounds) addresses and are issued unconditionally, the
  // values past the end being masked afterwards, so that each batch costs one round trip.
  {
    PhaseA& A = sh.x.a;
    const int CK = chunks * K;
    auto merge_row = [&](auto jm_tag, int i) __attribute__((always_inline)) {
      constexpr int JM = decltype(jm_tag)::value;   // 64-entry slices of the row's lists
      const uint64_t* rc = cand + ((size_t)b * D + i) * CK;
      uint64_t v[JM];
#pragma unroll
      for (int j = 0; j < JM; ++j) {
        const int e = j * kWave + lane;
        const uint64_t x = rc[min(e, CK - 1)];
        v[j] = e < CK ? x : 0ull;
      }
      const uint64_t hx = rc[(size_t)min(lane, chunks - 1) * K];
      const uint64_t head = lane < chunks ? hx : 0ull;
      // heads that beat this lane's head, read back from LDS eight at a time (every lane
      // reads the same address; the heads of lanes >= chunks are 0 and beat nothing)
      A.heads[wave][lane] = head;
      wave_fence();
      int beat = 0;
      for (int t0 = 0; t0 < chunks; t0 += 8) {
        uint64_t hv[8];
#pragma unroll
        for (int t = 0; t < 8; ++t) hv[t] = A.heads[wave][t0 + t];
#pragma unroll
        for (int t = 0; t < 8; ++t) beat += hv[t] > head ? 1 : 0;
      }
      const int nheads = __popcll(__ballot(head != 0ull));
      uint64_t T = 1ull;  // fewer non-empty chunks than K: every entry is a candidate
      if (nheads >= K) {
        const int tl = __ffsll((long long)__ballot(head != 0ull && beat == K - 1)) - 1;
        T = read_lane_u64(head, tl);
      }
      // compact the entries >= T (at most K*K of them) in order
      int total = 0;
#pragma unroll
      for (int j = 0; j < JM; ++j) {
        const uint64_t m = __ballot(v[j] >= T);
        const int pos = total + lanes_below(m);
        if (v[j] >= T && pos < kRowCap) A.rowc[wave][pos] = v[j];
        total += __popcll(m);
      }
      total = total < kRowCap ? total : kRowCap;
      wave_fence();
      const size_t orow = ((size_t)b * D + i) * K;
      // More than a wave's worth of candidates (flat rows): the K-th largest of them, T2,
      // by a descent over the key bits in which the candidates differ (the others are
      // common to all of them, so T2 has them too); the K entries >= T2 (keys are unique)
      // replace the candidate list.
      if (total > kWave) {   // uniform
        constexpr int JC = kRowCap / kWave;
        uint64_t cv[JC];
        uint64_t lor = 0ull, land = ~0ull;   // over this lane's candidates
#pragma unroll
        for (int j = 0; j < JC; ++j) {
          const int e = j * kWave + lane;
          const uint64_t x = A.rowc[wave][e];
          cv[j] = e < total ? x : 0ull;
          lor |= e < total ? x : 0ull;
          land &= e < total ? x : ~0ull;
        }
        const uint64_t gor = ((uint64_t)wave_or_u32((uint32_t)(lor >> 32)) << 32) |
                             wave_or_u32((uint32_t)lor);
        const uint64_t gand = ((uint64_t)wave_and_u32((uint32_t)(land >> 32)) << 32) |
                              wave_and_u32((uint32_t)land);
        const uint64_t diff = gor ^ gand;
        uint64_t T2 = gand & ~diff;
        for (uint64_t m = diff; m != 0ull;) {   // uniform
          const int bit = 63 - __clzll((long long)m);
          m &= ~(1ull << bit);
          const uint64_t c = T2 | (1ull << bit);
          int nc = 0;
#pragma unroll
          for (int j = 0; j < JC; ++j)
            if (j * kWave < total) nc += __popcll(__ballot(cv[j] >= c));
          if (nc >= K) T2 = c;
        }
        wave_fence();   // every lane has read the list before it is overwritten
        int kept = 0;
#pragma unroll
        for (int j = 0; j < JC; ++j) {
          const uint64_t m = __ballot(cv[j] >= T2);
          const int pos = kept + lanes_below(m);
          if (cv[j] >= T2) A.rowc[wave][pos] = cv[j];
          kept += __popcll(m);
        }
        total = kept;   // == K
        wave_fence();
      }
      // exact ranks of the (at most 64) candidates, one per lane, read back from LDS
      // eight at a time; the entry of rank r < K is the row's r-th candidate
      {
        const uint64_t mx = A.rowc[wave][lane];
        const uint64_t mine = lane < total ? mx : 0ull;
        int rank = 0;
        for (int t0 = 0; t0 < total; t0 += 8) {
          uint64_t rv[8];
#pragma unroll
          for (int t = 0; t < 8; ++t) {
            const uint64_t x = A.rowc[wave][t0 + t];
            rv[t] = t0 + t < total ? x : 0ull;
          }
#pragma unroll
          for (int t = 0; t < 8; ++t) rank += rv[t] > mine ? 1 : 0;
        }
        if (lane < total && rank < K) {
          sh.top[i][rank] = mine;
          o_tidx[orow + rank] = (int32_t)cand_index(mine);
          if (o_tval) o_tval[orow + rank] = value_from_key((uint32_t)(mine >> 32));
        }
      }
      for (int r = total + lane; r < K; r += kWave) {   // a row with fewer than K entries
        sh.top[i][r] = 0ull;
        o_tidx[orow + r] = -1;
        if (o_tval) o_tval[orow + r] = value_from_key(0u);
      }
      wave_fence();
      // Eq. 1 for this row (lane r < K): e_r, then c_r = e_r / Z with Z summed in rank order
      if (lane < K) {
        const uint64_t k = sh.top[i][lane];
        const double x = k ? (double)value_from_key((uint32_t)(k >> 32)) : (double)__uint_as_float(0x7FC00000u);
        double e;
        if (kind == TAPS_LOGITS) {
          const uint64_t k0 = sh.top[i][0];
          const double x0 = k0 ? (double)value_from_key((uint32_t)(k0 >> 32)) : x;
          e = spec_exp(beta * (x - x0));
        } else {
          e = x > 0.0 ? x : 0.0;
        }
        sh.e[i][lane] = e;
      }
      wave_fence();
      if (learned) {
        // learned scorer: LOG(Z) and the entropy LOG(Z) - S / Z of the row from the exact
        // sums of its integer partials (multiples of 2^-42); q_cond comes later
        const int zn = chunks * kZSub;
        const int64_t* zr = zpart + ((size_t)b * D + i) * zn;
        const int64_t* sr = spart + ((size_t)b * D + i) * zn;
        int64_t zp = 0, sp = 0;
        for (int c0 = lane; c0 < zn; c0 += kWave) {
          zp += zr[c0];
          sp += sr[c0];
        }
        const int64_t zi = wave_sum_i64(zp), si = wave_sum_i64(sp);
        if (lane == 0) {
          const double Z = (double)zi * 0x1p-42, S = (double)si * 0x1p-42;
          const double lz = zi > 0 ? spec_log(Z) : __longlong_as_double(0x7FF8000000000000ll);
          sh.lz[i] = lz;
          sh.ent[i] = lz - S / Z;
        }
      } else if (zpart) {
        // marginal scorer, logits (beta is 1): the full-vocabulary normaliser is the exact
        // sum of the row's integer partials (multiples of 2^-42)
        const int zn = chunks * kZSub;
        const int64_t* zr = zpart + ((size_t)b * D + i) * zn;
        int64_t zp = 0;
        for (int c0 = lane; c0 < zn; c0 += kWave) zp += zr[c0];
        const int64_t zi = wave_sum_i64(zp);
        const double Z = (double)zi * 0x1p-42;
        if (lane < K) sh.c[i][lane] = Z > 0.0 ? sh.e[i][lane] / Z : 0.0;
      } else if (kind == TAPS_PROBS && marginal) {
        // the probability itself (e = x if x > 0, else 0), clamped to 1
        if (lane < K) sh.c[i][lane] = fmin(sh.e[i][lane], 1.0);
      } else if (lane < K) {
        double Z = 0.0;
        for (int j = 0; j < K; ++j) Z = Z + sh.e[i][j];
        const bool ok = Z > 0.0 && Z <= 1.7976931348623157e308;
        sh.c[i][lane] = ok ? sh.e[i][lane] / Z : 0.0;
      }
    };
    // Two rows per wave, one per 32-lane half (row 2 pr + h in half h), for the common
    // shapes: K <= 8 (at most K*K <= 64 entries reach the threshold, two per lane), at
    // most 32 chunks (one head per lane) and 256 list entries.  Same steps and arithmetic
    // as merge_row; every instruction serves two rows, which halves the issue work of this
    // phase.
    auto merge_pair = [&](auto jm_tag, int pr) __attribute__((always_inline)) {
      constexpr int JM = decltype(jm_tag)::value;   // 32-entry slices of a row's lists
      const int h = lane >> 5, hl = lane & 31;
      const int i = 2 * pr + h;
      const bool rv = i < D;                        // a half past the last row idles
      const uint64_t* rc = cand + ((size_t)b * D + (rv ? i : D - 1)) * CK;
      uint64_t v[JM];
#pragma unroll
      for (int j = 0; j < JM; ++j) {
        const int e = j * 32 + hl;
        const uint64_t x = rc[min(e, CK - 1)];
        v[j] = rv && e < CK ? x : 0ull;
      }
      const uint64_t hx = rc[(size_t)min(hl, chunks - 1) * K];
      const uint64_t head = rv && hl < chunks ? hx : 0ull;
      // the normaliser partials of the marginal and learned scorers (at most 4 per lane):
      // loaded with the lists, since they do not depend on the merge
      const int zn = chunks * kZSub;
      int64_t zp = 0, sp = 0;
      if (zpart) {   // uniform
        const size_t zo = ((size_t)b * D + (rv ? i : D - 1)) * zn;
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int c0 = q * 32 + hl;
          const int64_t z = zpart[zo + min(c0, zn - 1)];
          zp += c0 < zn ? z : 0;
          if (learned) {
            const int64_t t = spart[zo + min(c0, zn - 1)];
            sp += c0 < zn ? t : 0;
          }
        }
      }
      uint64_t* hd = &A.heads[wave][h * 33];
      hd[hl] = head;
      wave_fence();
      int beat = 0;
      for (int t0 = 0; t0 < chunks; t0 += 8) {
        uint64_t hv[8];
#pragma unroll
        for (int t = 0; t < 8; ++t) hv[t] = hd[t0 + t];
#pragma unroll
        for (int t = 0; t < 8; ++t) beat += hv[t] > head ? 1 : 0;
      }
      // the K-th largest head of each half (fewer than K heads: every entry counts)
      const uint64_t nz = __ballot(head != 0ull);
      const uint64_t kth = __ballot(head != 0ull && beat == K - 1);
      uint64_t T0 = 1ull, T1 = 1ull;
      if (__popc((uint32_t)nz) >= K) T0 = read_lane_u64(head, __ffs((uint32_t)kth) - 1);
      if (__popc((uint32_t)(nz >> 32)) >= K)
        T1 = read_lane_u64(head, 31 + __ffs((uint32_t)(kth >> 32)));
      const uint64_t T = h ? T1 : T0;
      // compact each half's entries >= T (at most K*K <= 64) in order
      uint64_t* rw = &A.rowc[wave][h * 64];
      int total = 0;
#pragma unroll
      for (int j = 0; j < JM; ++j) {
        const bool keep = v[j] >= T;
        const uint64_t m = __ballot(keep);
        const uint32_t mlo = (uint32_t)m, mhi = (uint32_t)(m >> 32);
        const int pos = total + (int)__builtin_amdgcn_mbcnt_hi(h ? mhi : 0u,
                                                              __builtin_amdgcn_mbcnt_lo(h ? 0u : mlo, 0u));
        if (keep) rw[pos] = v[j];
        total += __popc(h ? mhi : mlo);
      }
      wave_fence();
      const int tmax = max(__builtin_amdgcn_readlane(total, 0), __builtin_amdgcn_readlane(total, 32));
      // exact ranks of the candidates (lane hl holds entries hl and 32 + hl of its half)
      const size_t orow = ((size_t)b * D + i) * K;
      {
        const uint64_t x0 = rw[hl], x1 = rw[32 + hl];
        const uint64_t c0 = hl < total ? x0 : 0ull, c1 = 32 + hl < total ? x1 : 0ull;
        int r0 = 0, r1 = 0;
        for (int t0 = 0; t0 < tmax; t0 += 8) {
          uint64_t rv8[8];
#pragma unroll
          for (int t = 0; t < 8; ++t) {
            const uint64_t x = rw[t0 + t];
            rv8[t] = t0 + t < total ? x : 0ull;
          }
#pragma unroll
          for (int t = 0; t < 8; ++t) r0 += rv8[t] > c0 ? 1 : 0;
          if (tmax > 32) {   // uniform
#pragma unroll
            for (int t = 0; t < 8; ++t) r1 += rv8[t] > c1 ? 1 : 0;
          }
        }
        if (rv && hl < total && r0 < K) {
          sh.top[i][r0] = c0;
          o_tidx[orow + r0] = (int32_t)cand_index(c0);
          if (o_tval) o_tval[orow + r0] = value_from_key((uint32_t)(c0 >> 32));
        }
        if (rv && 32 + hl < total && r1 < K) {
          sh.top[i][r1] = c1;
          o_tidx[orow + r1] = (int32_t)cand_index(c1);
          if (o_tval) o_tval[orow + r1] = value_from_key((uint32_t)(c1 >> 32));
        }
      }
      if (rv && total + hl < K) {   // a row with fewer than K entries
        const int r = total + hl;
        sh.top[i][r] = 0ull;
        o_tidx[orow + r] = -1;
        if (o_tval) o_tval[orow + r] = value_from_key(0u);
      }
      wave_fence();
      // Eq. 1 for each half's row (lane hl < K)
      if (rv && hl < K) {
        const uint64_t k = sh.top[i][hl];
        const double x = k ? (double)value_from_key((uint32_t)(k >> 32)) : (double)__uint_as_float(0x7FC00000u);
        double e;
        if (kind == TAPS_LOGITS) {
          const uint64_t k0 = sh.top[i][0];
          const double x0 = k0 ? (double)value_from_key((uint32_t)(k0 >> 32)) : x;
          e = spec_exp(beta * (x - x0));
        } else {
          e = x > 0.0 ? x : 0.0;
        }
        sh.e[i][hl] = e;
      }
      wave_fence();
      if (learned) {
        // learned scorer: LOG(Z) and the entropy LOG(Z) - S / Z of the row from the exact
        // sums of its integer partials (multiples of 2^-42); q_cond comes later
        const int64_t zi = half_sum_i64(zp), si = half_sum_i64(sp);
        if (rv && hl == 0) {
          const double Z = (double)zi * 0x1p-42, S = (double)si * 0x1p-42;
          const double lz = zi > 0 ? spec_log(Z) : __longlong_as_double(0x7FF8000000000000ll);
          sh.lz[i] = lz;
          sh.ent[i] = lz - S / Z;
        }
      } else if (zpart) {
        // marginal scorer, logits (beta is 1): the full-vocabulary normaliser is the exact
        // sum of the row's integer partials (multiples of 2^-42)
        const int64_t zi = half_sum_i64(zp);
        const double Z = (double)zi * 0x1p-42;
        if (rv && hl < K) sh.c[i][hl] = Z > 0.0 ? sh.e[i][hl] / Z : 0.0;
      } else if (rv && hl < K) {
        if (kind == TAPS_PROBS && marginal) {
          sh.c[i][hl] = fmin(sh.e[i][hl], 1.0);
        } else {
          double Z = 0.0;
          for (int j = 0; j < K; ++j) Z = Z + sh.e[i][j];
          const bool ok = Z > 0.0 && Z <= 1.7976931348623157e308;
          sh.c[i][hl] = ok ? sh.e[i][hl] / Z : 0.0;
        }
      }
    };
    if (K <= 8 && chunks <= 32 && CK <= 8 * 32) {
      for (int pr = wave; 2 * pr < D; pr += kWavesA) {
        if (CK <= 4 * 32) merge_pair(IntC<4>(), pr);
        else merge_pair(IntC<8>(), pr);
      }
    } else {
      for (int i = wave; i < D; i += kWavesA) {
        if (CK <= 4 * kWave) merge_row(IntC<4>(), i);
        else merge_row(IntC<16>(), i);
      }
    }
  }
  // Eq. 3 denominators lambda1 + lambda2 * depth
  if (tid <= D) sh.den[tid] = lambda1 + lambda2 * (double)tid;
  __syncthreads();
  // ---------------- learned scorer: q_cond table c3[i][parent rank][child rank] (all waves)
  extern __shared__ double s_c3[];
  double* c3 = learned ? s_c3 : nullptr;
  if (learned) {
    const int F = 2 * mlp.d + 3, d = mlp.d, h = mlp.h;
    const int edges = D * K * K, DK = D * K;
    // The scratch area (free until Phase C) holds, in order: the weights (W1, b1, w2 as
    // fp32), the embeddings of the root's token (slot 0) and of each candidate (slot
    // 1 + i*K + r; zeros for no token) at an odd row stride, each unit's three edge-feature
    // weights and its w2 widened to fp64 (so that the edges read them two at a time and
    // convert nothing), and per hidden unit k the parent part b1[k] + P_k of each possible
    // parent (0: the root, 1 + (i-1)*K + pr: the rank-pr candidate of row i-1) followed by
    // the child part C_k of each candidate, for a chunk of KC units at a time.  Each edge
    // then adds its five terms per unit.
    const LearnedLayout lay = learned_layout(D, K, d, h);
    float* Ws = reinterpret_cast<float*>(&sh.x);
    const int ES = lay.ES, np = lay.np, S = lay.S, KC = lay.KC;
    float* Es = Ws + lay.wsz;
    double* Wd = reinterpret_cast<double*>(Es + lay.esz);
    double* part = Wd + 4 * h;
    for (int j = tid; j < h * F; j += kThreadsA) Ws[j] = mlp.W1[j];
    for (int j = tid; j < h; j += kThreadsA) {
      const float w2j = mlp.w2[j];
      Ws[h * F + j] = mlp.b1[j];
      Ws[h * F + h + j] = w2j;
      Wd[4 * j] = (double)mlp.W1[j * F + 2 * d];
      Wd[4 * j + 1] = (double)mlp.W1[j * F + 2 * d + 1];
      Wd[4 * j + 2] = (double)mlp.W1[j * F + 2 * d + 2];
      Wd[4 * j + 3] = (double)w2j;
    }
    for (int j = tid; j < (DK + 1) * d; j += kThreadsA) {
      const int es = j / d, jj = j - es * d;
      int tok = -1;
      if (es == 0) {
        tok = mlp.root_token[b];
        if (tok >= mlp.vocab) tok = -1;   // outside the vocabulary: a zero embedding
      } else {
        const uint64_t kc = sh.top[(es - 1) / K][(es - 1) % K];
        if (kc) tok = (int)cand_index(kc);
      }
      Es[es * ES + jj] = tok >= 0 ? mlp.emb[(size_t)tok * d + jj] : 0.0f;
    }
    for (int ed = tid; ed < edges; ed += kThreadsA) {
      const int i = ed / (K * K), pr = (ed / K) % K, r = ed % K;
      c3[ed] = sh.top[i][r] && (i > 0 || pr == 0) ? (double)mlp.b2 : -INFINITY;
    }
    __syncthreads();
    for (int k0 = 0; k0 < h; k0 += KC) {
      const int kn = min(KC, h - k0);
      // the embedding sums, in index order from 0: one slot and eight units per thread
      // (units past the chunk are computed on a clamped unit and dropped)
      constexpr int U = 8;
      const int G = (kn + U - 1) / U;
      for (int t = tid; t < G * S; t += kThreadsA) {
        const int g = t / S, sl = t - g * S;
        const bool child = sl >= np;
        const float* e = Es + (child ? 1 + sl - np : sl) * ES;
        const float* w[U];
#pragma unroll
        for (int u = 0; u < U; ++u) w[u] = Ws + min(k0 + g * U + u, h - 1) * F + (child ? d : 0);
        double acc[U];
#pragma unroll
        for (int u = 0; u < U; ++u) acc[u] = 0.0;
        for (int j = 0; j < d; ++j) {
          const double ej = (double)e[j];
#pragma unroll
          for (int u = 0; u < U; ++u) acc[u] = acc[u] + (double)w[u][j] * ej;
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
          const int kk = g * U + u;
          if (kk < kn) part[kk * S + sl] = child ? acc[u] : (double)Ws[h * F + k0 + kk] + acc[u];
        }
      }
      __syncthreads();
      // each edge's logit over the chunk's units, four units at a time
      for (int ed = tid; ed < edges; ed += kThreadsA) {
        const int i = ed / (K * K), pr = (ed / K) % K, r = ed % K;
        const uint64_t kc = sh.top[i][r];
        if (!kc || (i == 0 && pr > 0)) continue;
        const double M = (double)value_from_key((uint32_t)(sh.top[i][0] >> 32));
        const double x = (double)value_from_key((uint32_t)(kc >> 32));
        const double lp = (x - M) - sh.lz[i];
        const double depth = (double)(i + 1), H = sh.ent[i];
        const int ps = i == 0 ? 0 : 1 + (i - 1) * K + pr, cs = np + i * K + r;
        double logit = c3[ed];
        for (int kk = 0; kk < kn; kk += 4) {
          double av[4], w2v[4];
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            const int k = min(kk + u, kn - 1);
            const double* w = Wd + 4 * (k0 + k);
            double a = part[k * S + ps] + part[k * S + cs];
            a = a + w[0] * depth;
            a = a + w[1] * lp;
            a = a + w[2] * H;
            av[u] = a > 0.0 ? a : 0.0;
            w2v[u] = w[3];
          }
#pragma unroll
          for (int u = 0; u < 4; ++u)
            if (kk + u < kn) logit = logit + w2v[u] * av[u];
        }
        c3[ed] = logit;
      }
      __syncthreads();
    }
    // sibling softmax of each parent's K logits, one child per thread: the terms EXP(l - max)
    // into the scratch area (the weights are no longer needed; D*K*K doubles fit), then the
    // rank-order sum and the quotients.  Row 0 has only the root as parent; its other parent
    // ranks take the root's entries.
    double* ex = reinterpret_cast<double*>(&sh.x);
    static_assert(sizeof(Scratch) >= kMaxLearnedEdges * sizeof(double), "terms fit the scratch");
    for (int t = tid; t < edges; t += kThreadsA) {
      const int pi = t / K, r = t - pi * K;
      if (pi < K && pi > 0) continue;
      const double* lg = c3 + (size_t)pi * K;
      double m = -INFINITY;
      for (int j = 0; j < K; ++j) m = fmax(m, lg[j]);   // NaN logits ignored
      ex[t] = spec_exp(lg[r] - m);
    }
    __syncthreads();
    for (int t = tid; t < edges; t += kThreadsA) {
      const int pi = t / K, r = t - pi * K;
      const double* e = ex + (size_t)(pi < K ? 0 : pi) * K;
      double Z = 0.0;
      for (int j = 0; j < K; ++j) Z = Z + e[j];
      const bool ok = Z > 0.0 && Z <= 1.7976931348623157e308;
      c3[t] = ok ? e[r] / Z : 0.0;
    }
    __syncthreads();
  }
  // The selection proper runs on the first four waves.  The other waves end here; a
  // workgroup barrier waits only for the waves that have not ended, so the barriers
  // below synchronize the remaining four.
  if (wave >= kWaves) return;

  // ---------------- Phase C: depth-by-depth expansion with a safe pruning bin
  // floor(n / K) for 0 <= n < 2^20 as a high multiply by ceil(2^32 / K): the error term
  // n (ceil(2^32/K) - 2^32/K) / 2^32 < 2^-12 never reaches the next integer
  const uint32_t kmul = K > 1 ? (uint32_t)((0x100000000ull + (uint64_t)K - 1) / (uint64_t)K) : 0u;
  auto divK = [&](int v) { return K > 1 ? (int)__umulhi((uint32_t)v, kmul) : v; };
  Level& L = sh.x.l;
  for (int j = tid; j < kBins; j += kThreads) L.hist[j] = 0;
  if (tid < kCoarse) L.chist[tid] = 0;
  if (tid == 0) {
    L.q[0] = 1.0;
    L.u[0] = ubits(1.0 / sh.den[0]);
    L.meta[0] = (0xFFFF << 16) | 0;
  }
  __syncthreads();
  // uniform state: stored nodes [p0, p1) form the current depth, base nodes are stored
  int parity = 0;
  int p0 = 0, p1 = 1, base = 1, bstar = 0;
  bool bstar_due = false;   // the histograms hold a level whose pruning bin is not taken yet
  bool fallback = false;
  for (int d = 0; d < D && N > 1; ++d) {
    const int items = (p1 - p0) * K;
    if (items == 0) break;
    const double den1 = sh.den[d + 1];
    // the level's items in chunks of up to 4 per thread, each thread taking contiguous
    // items so that the stored order stays (parent, rank)
    for (int c0 = 0; c0 < items; c0 += 4 * kThreads) {
      const int citems = min(items - c0, 4 * kThreads);
      const int per = (citems + kThreads - 1) / kThreads;
      // evaluate this thread's candidates once: child r of stored node p at depth d
      double qv[4], uv[4];
      int mv[4], bv[4];
      bool okv[4];
      int cnt = 0;
      const int it0 = c0 + tid * per;
      const int q0 = divK(it0);
      // items past this thread's count are evaluated too (clamped parent index, so every
      // load is in bounds and the loads and fp64 arithmetic of all items overlap) and
      // masked; a chunk of at most one item per thread evaluates one
      auto eval = [&](auto ni_tag) __attribute__((always_inline)) {
        constexpr int NI = decltype(ni_tag)::value;
        int pp = p0 + q0, rr = it0 - q0 * K;   // (parent, rank) of the first item
        uint64_t puv[NI];
        double qpv[NI], crv[NI];
        int pv[NI], rv[NI];
#pragma unroll
        for (int k = 0; k < NI; ++k) {
          const int p = pp, r = rr;
          if (++rr == K) { rr = 0; ++pp; }
          const int pc = min(p, p1 - 1);
          puv[k] = L.u[pc];
          qpv[k] = L.q[pc];
          crv[k] = c3 ? c3[(d * K + (L.meta[pc] & 0xFF)) * K + r] : sh.c[d][r];
          pv[k] = p;
          rv[k] = r;
        }
        // the pruning bin of the previous level, read from its histograms while the
        // loads above are in flight
        if (bstar_due) {   // uniform
          bstar = find_bstar(L, N);
          bstar_due = false;
        }
#pragma unroll
        for (int k = 0; k < NI; ++k) {
          const int it = it0 + k;
          const int p = pv[k], r = rv[k];
          const uint64_t pu = puv[k];
          const double q = qpv[k] * crv[k];
          const double u = q / den1;
          const int bn = ubin(u);
          // non-short-circuit: no branch may separate a load from the others
          okv[k] = (k < per) & (it < c0 + citems) &
                   (ubin(__longlong_as_double((long long)pu)) >= bstar) & (u > tau) & (bn >= bstar);
          qv[k] = q;
          uv[k] = u;
          bv[k] = bn;
          mv[k] = (p << 16) | ((d + 1) << 8) | r;
          cnt += okv[k] ? 1 : 0;
        }
#pragma unroll
        for (int k = NI; k < 4; ++k) okv[k] = false;
      };
      if (per == 1) eval(IntC<1>());
      else eval(IntC<4>());
      int total;
      const int pre = block_prefix(cnt, sh.wsum, parity, total);
      if (base + total > kCap) {       // uniform: the expansion outgrows LDS
        fallback = true;
        break;
      }
      int pos = base + pre;
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        if (okv[k]) {
          L.q[pos] = qv[k];
          L.u[pos] = ubits(uv[k]);
          L.meta[pos] = mv[k];
          atomicAdd(&L.hist[bv[k]], 1);
          atomicAdd(&L.chist[bv[k] >> 4], 1);
          ++pos;
        }
      }
      base += total;
      // once N-1 nodes are stored, the pruning bin can rise after every chunk, also in
      // the middle of a level: every node below it is beaten by N-1 stored nodes
      if (base >= N - 1 && c0 + 4 * kThreads < items) {   // uniform
        __syncthreads();   // the chunk's histogram counts are complete
        bstar = find_bstar(L, N);
      }
    }
    if (fallback) break;
    __syncthreads();   // the level's nodes and histogram counts are complete
    p0 = p1;
    p1 = base;
    bstar_due = base >= N - 1;
  }
  if (bstar_due && !fallback) bstar = find_bstar(L, N);
  int n;
  if (!fallback) {
    // ---- final cut: keep bins > b*; members of bin b* compete for the places left.
    // Thread t owns the stored nodes t*per .. t*per + per - 1 (per <= kCap / kThreads);
    // bit k of a mask below stands for its node t*per + k.
    const int tot = base;
    const int per = (tot + kThreads - 1) / kThreads;
    const int j0 = tid * per;
    const int jn = min(per, tot - j0);   // nodes this thread owns (may be <= 0)
    uint32_t amask = 0u, bmask = 0u;     // bins > b* (the root counts here), bin b*
    for (int k = 0; k < jn; ++k) {
      const int j = j0 + k;
      const int bn = ubin(__longlong_as_double((long long)L.u[j]));
      if (j == 0 || bn > bstar) amask |= 1u << k;
      else if (bn == bstar) bmask |= 1u << k;
    }
    const int above = __popc(amask) - (j0 == 0 && jn > 0 ? 1 : 0), inb = __popc(bmask);
    // both counts in one prefix: each total stays below 2^16
    int tot2;
    const int pre2 = block_prefix(above | (inb << 16), sh.wsum, parity, tot2);
    const int c_hi = tot2 & 0xFFFF, c_b = tot2 >> 16;
    const int room = N - 1 - c_hi;   // places left for members of bin b*
    uint32_t kmask = amask | bmask;
    if (c_b > room) {                // uniform: the members of bin b* are ranked
      // The members' utility bits go to a list in stored order, so that a member's list
      // position orders equal utilities like its stored index, i.e. like (depth, rank
      // path).  A member is kept if fewer than `room` members beat it under (u desc,
      // position asc).  One member per thread, all threads reading the same list entries;
      // the losers are marked in a bitmask (over the histogram, no longer needed).
      int mpos = pre2 >> 16;
      for (uint32_t m = bmask; m; m &= m - 1) L.mkey[mpos++] = L.u[j0 + __ffs(m) - 1];
      for (int w = tid; w < (c_b + 31) / 32; w += kThreads) L.hist[w] = 0;
      __syncthreads();
      for (int m = tid; m < c_b; m += kThreads) {
        const uint64_t um = L.mkey[m];
        int rank = 0;
        for (int k0 = 0; k0 < c_b; k0 += 8) {
          uint64_t uk[8];
#pragma unroll
          for (int t = 0; t < 8; ++t) uk[t] = L.mkey[min(k0 + t, c_b - 1)];
#pragma unroll
          for (int t = 0; t < 8; ++t) {
            const int k = k0 + t;
            rank += (k < c_b && (uk[t] > um || (uk[t] == um && k < m))) ? 1 : 0;
          }
        }
        if (rank >= room) atomicOr(&L.hist[m >> 5], (int)(1u << (m & 31)));
      }
      __syncthreads();
      int mp = pre2 >> 16;
      for (uint32_t m = bmask; m; m &= m - 1, ++mp)
        if ((L.hist[mp >> 5] >> (mp & 31)) & 1) kmask &= ~(1u << (__ffs(m) - 1));
    }
    // breadth-first compaction: stored order is already (depth, rank path)
    int total;
    const int pos0 = block_prefix(__popc(kmask), sh.wsum, parity, total);
    {
      int pos = pos0;
      for (int k = 0; k < jn; ++k) {
        const bool kp = (kmask >> k) & 1u;
        L.newidx[j0 + k] = kp ? pos : -1;
        pos += kp ? 1 : 0;
      }
    }
    __syncthreads();
    n = total;
    {
      int pos = pos0;
      for (uint32_t m = kmask; m; m &= m - 1) {
        const int j = j0 + __ffs(m) - 1;
        const size_t g = (size_t)b * N + pos++;
        const int meta = L.meta[j];
        const int dj = (meta >> 8) & 0xFF, rj = meta & 0xFF, pj = meta >> 16;
        o_parent[g] = j == 0 ? -1 : L.newidx[pj];
        o_depth[g] = dj;
        o_rank[g] = j == 0 ? -1 : rj;
        o_token[g] = j == 0 ? -1 : (int32_t)cand_index(sh.top[dj - 1][rj]);
        o_q[g] = L.q[j];
      }
    }
  } else {
    __syncthreads();
    n = select_sequential<SLOTS>(sh, c3, D, K, N, tau);
    Seq& S = sh.x.s;
    for (int j = tid; j < n; j += kThreads) {
      const size_t g = (size_t)b * N + S.order[j];
      o_parent[g] = j == 0 ? -1 : S.order[S.par[j]];
      o_depth[g] = S.depth[j];
      o_rank[g] = S.rank[j];
      o_token[g] = j == 0 ? -1 : (int32_t)cand_index(sh.top[S.depth[j] - 1][S.rank[j]]);
      o_q[g] = S.q[j];
    }
  }
  // ---------------- Phase D: pad the unused slots
  for (int j = n + tid; j < N; j += kThreads) {
    const size_t g = (size_t)b * N + j;
    o_parent[g] = -1; o_depth[g] = -1; o_rank[g] = -1; o_token[g] = -1; o_q[g] = 0.0;
  }
  if (tid == 0) o_n[b] = n;
}

// Marginal scorer, logits: per (row, chunk) the integer partial of the full-vocabulary
// normaliser, sum over the chunk's entries of rint(2^42 * EXP(x_j - M)), where M is the
// row maximum (the largest chunk head the top-K pass wrote).  Integer sums are exact, so
// the order of the additions (here, and of the partials in the selection) does not enter.
// Grid: rows * chunks workgroups of 256 threads, the chunking of the top-K pass.
template <int DT>
__global__ __launch_bounds__(256) void marginal_z_kernel(const void* __restrict__ marg,
                                                         int vocab, int K, int chunk_len,
                                                         int chunks,
                                                         const uint64_t* __restrict__ cand,
                                                         int64_t* __restrict__ zpart,
                                                         int64_t* __restrict__ spart) {
  __shared__ double s_M;
  __shared__ int64_t s_w[4], s_s[4];
  const int row = blockIdx.x / (chunks * kZSub);
  const int part = blockIdx.x - row * (chunks * kZSub);   // chunk * kZSub + sub-range
  const int chunk = part / kZSub;
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
  if (wave == 0) {
    uint64_t h = 0ull;
    for (int c = lane; c < chunks; c += kWave) {
      const uint64_t x = cand[((size_t)row * chunks + c) * K];
      h = x > h ? x : h;
    }
    h = wave_max_u64(h);
    if (lane == 0) s_M = (double)value_from_key(h ? (uint32_t)(h >> 32) : 0u);
  }
  __syncthreads();
  const double M = s_M;
  const int sub_len = chunk_len / kZSub;
  const int start = chunk * chunk_len + (part - chunk * kZSub) * sub_len;
  const int end = min(vocab, start + sub_len);
  // The terms are integers (multiples of 2^-42 scaled by 2^42) below 2^42 in magnitude,
  // and a thread adds at most 64 of them, so fp64 holds its sums exactly; they become
  // int64 once per thread.
  double accd = 0.0, accsd = 0.0;
  // four elements per thread at a time (clamped loads, masked terms) so that their
  // exponentials overlap; the exact sums do not depend on the order
  for (int e0 = start + tid; e0 < end; e0 += 4 * 256) {
    double xv[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int e = min(e0 + j * 256, end - 1);
      if (DT == TAPS_BF16) {
        const uint16_t u = ((const uint16_t*)marg)[(size_t)row * vocab + e];
        xv[j] = (double)__uint_as_float((uint32_t)u << 16);
      } else {
        xv[j] = (double)((const float*)marg)[(size_t)row * vocab + e];
      }
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      if (e0 + j * 256 >= end) continue;
      const double dx = xv[j] - M;
      const double t = spec_exp(dx);
      accd += rint(t * 0x1p42);
      // the entropy's sum (learned scorer): t (x - M) on the same grid, 0 where t is 0
      if (spart) accsd += t > 0.0 ? rint((t * dx) * 0x1p42) : 0.0;
    }
  }
  const int64_t acc = wave_sum_i64((int64_t)accd);
  const int64_t accs = wave_sum_i64((int64_t)accsd);
  if (lane == 0) {
    s_w[wave] = acc;
    s_s[wave] = accs;
  }
  __syncthreads();
  if (tid == 0) {
    zpart[(size_t)row * chunks * kZSub + part] = s_w[0] + s_w[1] + s_w[2] + s_w[3];
    if (spart) spart[(size_t)row * chunks * kZSub + part] = s_s[0] + s_s[1] + s_s[2] + s_s[3];
  }
}

}  // namespace

double spec_exp_host(double t) { return spec_exp(t); }

hipError_t launch_marginal_z(const void* marg, int dtype, int rows, int vocab, int K,
                             const TopkPlan& plan, const uint64_t* cand, int64_t* zpart,
                             int64_t* spart, hipStream_t s) {
  if (rows <= 0) return hipSuccess;
  const dim3 grid((unsigned)(rows * plan.chunks * kZSub)), block(256);
  if (dtype == TAPS_BF16)
    marginal_z_kernel<TAPS_BF16><<<grid, block, 0, s>>>(marg, vocab, K, plan.chunk_len,
                                                        plan.chunks, cand, zpart, spart);
  else
    marginal_z_kernel<TAPS_FP32><<<grid, block, 0, s>>>(marg, vocab, K, plan.chunk_len,
                                                        plan.chunks, cand, zpart, spart);
  return hipGetLastError();
}

int learned_chunk_units(int D, int K, int d, int h) { return learned_layout(D, K, d, h).KC; }

hipError_t launch_select(const void* /*marg*/, const taps_select_params& p, const TopkPlan& plan,
                         const uint64_t* cand, const int64_t* zpart, const int64_t* spart,
                         const taps_tree& out, hipStream_t s) {
  dim3 grid((unsigned)p.batch), block(kThreadsA);
  const int slots = (p.budget + kWave - 1) / kWave;
  const int marginal = p.scorer == TAPS_SCORER_MARGINAL;
  ScorerArgs mlp{};
  size_t dyn = 0;
  if (p.scorer == TAPS_SCORER_LEARNED) {
    const taps_scorer_mlp& w = *p.mlp;
    mlp = ScorerArgs{w.emb, w.W1, w.b1, w.w2, w.b2, w.root_token, w.emb_dim, w.hidden, p.vocab};
    dyn = (size_t)p.block * p.K * p.K * sizeof(double);
  }
#define TAPS_SEL_L(SL, LR)                                                                    \
  do {                                                                                        \
    if (dyn && hipFuncSetAttribute((const void*)select_kernel<SL, LR>,                        \
                                   hipFuncAttributeMaxDynamicSharedMemorySize,                \
                                   (int)dyn) != hipSuccess)                                    \
      return hipErrorInvalidValue;                                                            \
    select_kernel<SL, LR><<<grid, block, dyn, s>>>(                                           \
        p.block, p.K, p.budget, p.kind, p.lambda1, p.lambda2, p.tau, p.beta, plan.chunks,     \
        marginal, cand, zpart, spart, mlp, out.parent, out.token, out.depth, out.rank,        \
        out.q_reach, out.n_nodes, out.topk_idx, out.topk_val);                                \
  } while (0)
#define TAPS_SEL(SL)                                                                          \
  do {                                                                                        \
    if (spart) TAPS_SEL_L(SL, true);                                                          \
    else TAPS_SEL_L(SL, false);                                                               \
  } while (0)
  static_assert(TAPS_MAX_BUDGET <= 8 * kWave, "at most eight frontier slots per lane");
  switch (slots) {
    case 1: TAPS_SEL(1); break;
    case 2: TAPS_SEL(2); break;
    case 3:
    case 4: TAPS_SEL(4); break;
    default: TAPS_SEL(8); break;
  }
#undef TAPS_SEL
#undef TAPS_SEL_L
  return hipGetLastError();
}

}  // namespace taps
