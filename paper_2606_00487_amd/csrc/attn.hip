// Tree-masked verification attention (Sec. 4.1 Stage 3; Sec. 4.3): each selected node
// attends to every cached context row of its request and to the tree rows of its
// ancestors and itself.
//
// bf16 path, split-KV flash attention on MFMA (gfx950 v_mfma_f32_32x32x16_bf16):
//   * one workgroup = (request, KV head, query-row tile, key split); the query rows of a
//     KV head are the tree nodes x the G query heads that share it, a dense tile;
//   * S^T = K Q^T: A = a 32-key block of K (LDS), B = Q^T (registers), so every lane
//     owns one query column and the row max needs one exchange between lane halves;
//   * O^T += V^T P^T: B = P^T comes straight from the S^T accumulators (converted to
//     bf16); the key order inside the MFMA k-dimension follows the accumulator layout,
//     and V is staged transposed in LDS in that order;
//   * K and V tiles are XOR-swizzled in LDS so the 16-byte reads of a wave hit distinct
//     banks;
//   * the ancestor-or-self bitmask of every node is rebuilt from parent pointers when a
//     split reaches the tree rows; keys beyond the split or outside the mask get -inf;
//   * fp32 online softmax in base 2; each split writes unnormalised O, its running max
//     and its sum; a second kernel combines the splits and rounds to bf16.
// fp32 path: a plain VALU kernel, one workgroup per (request, node, query head).
#include <cstdio>
#include <cstdlib>

#include "common.h"

namespace taps {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kThreads = 256;
constexpr int kWavesA = 4;
constexpr int kKT = 64;  // keys per tile
constexpr float kLog2e = 1.4426950408889634f;


// word w (0..3) of a 256-bit mask held in registers, without dynamic register indexing
__device__ inline uint64_t mask_word(const uint64_t (&a)[4], int w) {
  const uint64_t lo = (w & 1) ? a[1] : a[0];
  const uint64_t hi = (w & 1) ? a[3] : a[2];
  return (w & 2) ? hi : lo;
}

// ancestor-or-self mask of node i from parent pointers (a parent outside [0, node)
// ends the walk); par(j) reads the parent of node j
template <typename F>
__device__ inline void ancestor_mask(int i, F par, uint64_t (&a)[4]) {
  a[0] = a[1] = a[2] = a[3] = 0ull;
  int cur = i;
  for (;;) {
    const uint64_t bit = 1ull << (cur & 63);
    const int w = cur >> 6;
    a[0] |= w == 0 ? bit : 0ull;
    a[1] |= w == 1 ? bit : 0ull;
    a[2] |= w == 2 ? bit : 0ull;
    a[3] |= w == 3 ? bit : 0ull;
    const int p = par(cur);
    if (p < 0 || p >= cur) break;
    cur = p;
  }
}

// 64 keys of the 256-bit ancestor-or-self mask a[], starting at bit t0 (t0 may be negative:
// bits below 0 read as 0)
__device__ inline uint64_t mask_window(const uint64_t (&a)[4], int t0) {
  if (t0 <= -64 || t0 >= 256) return 0ull;
  if (t0 < 0) return a[0] << (-t0);
  const int w = t0 >> 6, sh = t0 & 63;
  const uint64_t lo = mask_word(a, w);
  const uint64_t hi = w < 3 ? mask_word(a, w + 1) : 0ull;
  return sh ? (lo >> sh) | (hi << (64 - sh)) : lo;
}

// bits j of a 64-bit window for j < 64 (0 for j <= 0, all ones for j >= 64)
__device__ inline uint64_t low_bits(int j) {
  return j <= 0 ? 0ull : (j >= 64 ? ~0ull : ((1ull << j) - 1ull));
}

typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;
typedef __attribute__((address_space(3))) void lds_void;

// s_waitcnt that waits until at most `n` vector-memory operations are outstanding
// (expcnt and lgkmcnt left at their maxima, i.e. not waited on)
#define TAPS_WAIT_VMCNT(n) \
  __builtin_amdgcn_s_waitcnt(((n) & 0xF) | ((((n) >> 4) & 3) << 14) | (7 << 4) | (15 << 8))

typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;

// permutation of a key row's low three bits that XORs its 16-byte chunks: the 8 rows a
// K read touches at once, and the 4 rows x 2 chunk pairs a transposing V read touches
// at once, land on distinct LDS banks
__device__ inline int kswz(int r) { return ((r & 3) << 1) | ((r >> 2) & 1); }

// QB: 32-row query blocks per wave; WK: key groups (each iteration stages WK tiles, wave
// group kg = wave / 4 works on tile kg; the groups merge their results in LDS at the end).
// K and V tiles go from global memory straight into LDS (16 bytes per lane), row-major
// with the 16-byte chunks of key row r XOR-permuted by kswz(r); two stages alternate so
// the next iteration's tiles load while the current ones are used.  V^T operands are
// read with the transposing LDS read: in each 16-lane group, lane i gets element i % 4
// of the 8 bytes read by lanes 4t + i/4 (t = 0..3), i.e. 4 consecutive keys at its d.
// The grid is one-dimensional: the query-row tiles of one (request, KV head, split) get
// block ids that differ by multiples of 8, so they run on the same XCD and share its L2.
template <int QB, int WK, int HD>
__global__ __launch_bounds__(256 * WK) void attn_bf16_kernel(
    const uint16_t* __restrict__ Q, const uint16_t* __restrict__ Kc,
    const uint16_t* __restrict__ Vc, const int64_t* __restrict__ offp,
    const int32_t* __restrict__ ctxp, const int32_t* __restrict__ parentp,
    const int32_t* __restrict__ nnp, int N, int Hq, int Hkv, int max_ctx, float scale_log2,
    int split_len, int splits, int mtiles, int pairs, int mrows_pad, float* __restrict__ wsO,
    float2* __restrict__ wsML) {
  constexpr int NT = 256 * WK;
  constexpr int NW = 4 * WK;
  constexpr int ROWB = HD * 2;        // bytes per K/V row
  constexpr int MT = 4 * 32 * QB;     // query rows per workgroup
  constexpr int NDB = HD / 32;        // 32-row blocks of O^T
  constexpr int NKK = HD / 16;        // MFMA k-steps over head_dim
  constexpr int TILEB = kKT * ROWB;   // bytes of one staged K (or V) tile
  constexpr int STAGEB = 2 * WK * TILEB;  // K and V tiles of the WK key groups
  constexpr int BLK = kWave * 16;     // bytes one wave writes per direct load
  constexpr int LPW = STAGEB / BLK / NW;  // direct loads per wave per stage
  constexpr int XBYTES = 4 * QB * NDB * 16 * 64 * 4;  // key-group exchange of O
  constexpr int SBYTES = (WK > 1 && XBYTES > 2 * STAGEB) ? XBYTES : 2 * STAGEB;
  static_assert(STAGEB % (BLK * NW) == 0, "stage must split evenly over the waves");
  static_assert(LPW <= 8, "direct loads per wave");
  __shared__ __attribute__((aligned(16))) unsigned char s_raw[SBYTES];
  __shared__ uint64_t s_anc[TAPS_MAX_BUDGET][4];
  __shared__ int s_par[TAPS_MAX_BUDGET];
  __shared__ float2 s_ml[WK > 1 ? 4 * QB * 64 : 1];

  // ---- which (request, KV head, split, row tile) this workgroup owns
  const int xcd = blockIdx.x & 7, slot = blockIdx.x >> 3;
  const int mt = slot % mtiles, pair = (slot / mtiles) * 8 + xcd;
  if (pair >= pairs) return;
  const int split = pair % splits, bg = pair / splits;
  const int b = bg / Hkv, g = bg - (bg / Hkv) * Hkv;
  const int G = Hq / Hkv;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int rg = wave & 3, kg = wave >> 2;
  const int l32 = lane & 31, hl = lane >> 5;

  const int ctx = min(max(ctxp[b], 0), max_ctx);
  const int n = min(max(nnp[b], 0), N);
  const int R = ctx + n;
  const int k_begin = split * split_len;
  const int k_end = min(R, k_begin + split_len);
  const int row0 = mt * MT;
  if (k_begin >= k_end || row0 >= n * G) return;
  const int64_t kv0 = offp[b];
  const size_t row_stride = (size_t)Hkv * HD;  // elements between consecutive cache rows
  const uint16_t* kbase = Kc + (size_t)kv0 * row_stride + (size_t)g * HD;
  const uint16_t* vbase = Vc + (size_t)kv0 * row_stride + (size_t)g * HD;

  // ---- per-lane pieces of the direct loads: block j of this wave covers 4 key rows
  int ld_row[LPW], ld_off[LPW];   // row within the stage's tile, element offset in the row
#pragma unroll
  for (int j = 0; j < LPW; ++j) {
    const int byte = (wave * LPW + j) * BLK + lane * 16;
    const int within = byte % (WK * TILEB);
    const int t = within / TILEB;
    const int rb = within - t * TILEB;
    const int kr = rb / ROWB;
    const int pc = (rb - kr * ROWB) / 16;
    ld_row[j] = t * kKT + kr;
    ld_off[j] = (pc ^ kswz(kr)) * 8;
  }
  auto issue_stage = [&](int stage, int base) {
    unsigned char* sb = s_raw + stage * STAGEB;
    const bool full = base + kKT * WK <= k_end;
#pragma unroll
    for (int j = 0; j < LPW; ++j) {
      const int blk = wave * LPW + j;
      const bool isv = blk * BLK >= WK * TILEB;   // uniform per wave and j
      int key = base + ld_row[j];
      if (!full) key = key < k_end ? key : k_begin;   // a real row; masked out later
      const uint16_t* src = (isv ? vbase : kbase) + (size_t)key * row_stride + ld_off[j];
      __builtin_amdgcn_global_load_lds((const void*)src, (lds_void*)(sb + blk * BLK), 16, 0, 0);
    }
  };
  constexpr int STEP = kKT * WK;
  issue_stage(0, k_begin);   // the first tiles load while the queries and masks are set up

  // ---- queries of this lane (B operand of S^T = K Q^T)
  bf16x8 q[QB][NKK];
  int qnode[QB];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    int qr = row0 + rg * 32 * QB + qb * 32 + l32;
    qr = min(qr, N * G - 1);
    const int node = qr / G, hq = g * G + (qr - node * G);
    qnode[qb] = node;
    const uint16_t* qp = Q + (((size_t)b * N + node) * Hq + hq) * HD;
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk) q[qb][kk] = *(const bf16x8*)(qp + kk * 16 + hl * 8);
  }

  // ---- ancestor masks, only when this split reaches the tree rows
  uint64_t anc[QB][4];
  if (k_end > ctx) {
    for (int i = tid; i < n; i += NT) s_par[i] = parentp[(size_t)b * N + i];
    __syncthreads();
    for (int i = tid; i < n; i += NT) {
      uint64_t a[4];
      ancestor_mask(i, [&](int j) { return s_par[j]; }, a);
#pragma unroll
      for (int w = 0; w < 4; ++w) s_anc[i][w] = a[w];
    }
    __syncthreads();
#pragma unroll
    for (int qb = 0; qb < QB; ++qb)
#pragma unroll
      for (int w = 0; w < 4; ++w) anc[qb][w] = qnode[qb] < n ? s_anc[qnode[qb]][w] : 0ull;
  } else {
#pragma unroll
    for (int qb = 0; qb < QB; ++qb)
#pragma unroll
      for (int w = 0; w < 4; ++w) anc[qb][w] = 0ull;
  }

  // ---- per-lane LDS read offsets (constant over iterations)
  // K: key row l32 (+32 per key block), chunk (2kk + hl) ^ kswz(l32)
  const int fk = kswz(l32);
  int koff[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) koff[j] = l32 * ROWB + 32 * (j ^ (fk >> 1)) + 16 * (hl ^ (fk & 1));
  // V^T: lanes 4t + q of each 16-lane group read row 4*hl + t, 8 bytes at d = 16*g16 + 4*q
  const int g16 = (lane >> 4) & 1, tq = (lane & 15) >> 2, qq = lane & 3;
  const int fv = kswz(4 * hl + tq);
  int voff[2];
#pragma unroll
  for (int j = 0; j < 2; ++j)
    voff[j] = (4 * hl + tq) * ROWB + 8 * (qq & 1) + 16 * ((g16 * 2 + (qq >> 1)) ^ (fv & 3)) +
              64 * (j ^ (fv >> 2));

  f32x16 o[NDB][QB];
#pragma unroll
  for (int db = 0; db < NDB; ++db)
#pragma unroll
    for (int qb = 0; qb < QB; ++qb)
#pragma unroll
      for (int v = 0; v < 16; ++v) o[db][qb][v] = 0.f;
  float m_ref[QB], l_run[QB];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) { m_ref[qb] = -INFINITY; l_run[qb] = 0.f; }

  int stage = 0;
  for (int base = k_begin; base < k_end; base += STEP, stage ^= 1) {
    const bool more = base + STEP < k_end;
    if (more) {
      issue_stage(stage ^ 1, base + STEP);
      TAPS_WAIT_VMCNT(LPW);          // this stage's loads are done, the next may fly
    } else {
      TAPS_WAIT_VMCNT(0);
    }
    __builtin_amdgcn_s_barrier();
    const int k0 = base + kg * kKT;
    if (k0 < k_end) {
      const unsigned char* tk = s_raw + stage * STAGEB + kg * TILEB;
      const unsigned char* tv = s_raw + stage * STAGEB + WK * TILEB + kg * TILEB;
      // ---- S^T = K Q^T for the two 32-key blocks
      f32x16 s[2][QB];
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
        for (int qb = 0; qb < QB; ++qb)
#pragma unroll
          for (int v = 0; v < 16; ++v) s[kb][qb][v] = 0.f;
#pragma unroll
        for (int kk = 0; kk < NKK; ++kk) {
          const bf16x8 a = *(const bf16x8*)(tk + kb * 32 * ROWB + 32 * (kk & ~3) + koff[kk & 3]);
#pragma unroll
          for (int qb = 0; qb < QB; ++qb)
            s[kb][qb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, q[qb][kk], s[kb][qb], 0, 0, 0);
        }
      }
      // ---- mask (only tiles that reach the tree rows or the split end), online softmax
      const bool need_mask = k0 + kKT > ctx || k0 + kKT > k_end;
      float nrefv[QB];
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) {
        if (need_mask) {
          uint64_t A = (low_bits(ctx - k0) | mask_window(anc[qb], k0 - ctx)) & low_bits(k_end - k0);
          A >>= 4 * hl;   // this lane's keys are kb*32 + 8*(v/4) + 4*hl + v%4
          const uint32_t mlo = (uint32_t)A, mhi = (uint32_t)(A >> 32);
#pragma unroll
          for (int kb = 0; kb < 2; ++kb)
#pragma unroll
            for (int v = 0; v < 16; ++v) {
              const uint32_t word = kb ? mhi : mlo;
              const bool ok = (word >> (8 * (v >> 2) + (v & 3))) & 1u;
              s[kb][qb][v] = ok ? s[kb][qb][v] : -INFINITY;
            }
        }
        float mx = -INFINITY;
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int v = 0; v < 16; ++v) mx = fmaxf(mx, s[kb][qb][v]);
        mx = fmaxf(mx, __shfl_xor(mx, 32)) * scale_log2;   // scale > 0
        // move the reference max only when it is exceeded by more than 2^8
        const bool upd = mx > m_ref[qb] + 8.f;
        if (__ballot(upd)) {
          const float nref = upd ? mx : m_ref[qb];
          const float alpha = upd ? __builtin_amdgcn_exp2f(m_ref[qb] - nref) : 1.f;
          l_run[qb] *= alpha;
#pragma unroll
          for (int db = 0; db < NDB; ++db)
#pragma unroll
            for (int v = 0; v < 16; ++v) o[db][qb][v] *= alpha;
          m_ref[qb] = nref;
        }
        nrefv[qb] = m_ref[qb] == -INFINITY ? 0.f : -m_ref[qb];
      }
      // ---- P = exp2(scale*s - ref) and O^T += V^T P^T in four groups of 8 keys per lane
      // half: the exponentials of one group are independent of the MFMAs of the previous
      // group, so the two overlap.  V^T operands come from transposing reads of the
      // row-major V tile.
#pragma unroll
      for (int grp = 0; grp < 4; ++grp) {
        const int kb = grp >> 1, hf = grp & 1;
        bf16x8 pg[QB];
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) {
          float sum = 0.f;
#pragma unroll
          for (int t = 0; t < 8; ++t) {
            const float e = __builtin_amdgcn_exp2f(fmaf(s[kb][qb][hf * 8 + t], scale_log2, nrefv[qb]));
            sum += e;
            pg[qb][t] = (__bf16)e;
          }
          l_run[qb] += sum;
        }
#pragma unroll
        for (int db = 0; db < NDB; ++db) {
          const unsigned char* va = tv + (kb * 32 + 16 * hf) * ROWB + voff[db & 1] + 64 * (db & ~1);
          const bf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)va);
          const bf16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(va + 8 * ROWB));
          const bf16x8 a = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
#pragma unroll
          for (int qb = 0; qb < QB; ++qb)
            o[db][qb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pg[qb], o[db][qb], 0, 0, 0);
        }
      }
    }
    __builtin_amdgcn_s_barrier();    // the stage is free for the loads issued next iteration
  }

  float lsum[QB];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) lsum[qb] = l_run[qb] + __shfl_xor(l_run[qb], 32);

  // ---- merge the key groups through LDS (the stage buffers are free now)
  if (WK > 1) {
    float* xo = (float*)s_raw;
    if (kg == 1) {
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) {
#pragma unroll
        for (int db = 0; db < NDB; ++db)
#pragma unroll
          for (int v = 0; v < 16; ++v)
            xo[(((rg * QB + qb) * NDB + db) * 16 + v) * 64 + lane] = o[db][qb][v];
        s_ml[(rg * QB + qb) * 64 + lane] = make_float2(m_ref[qb], lsum[qb]);
      }
    }
    __syncthreads();
    if (kg != 0) return;
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      const float2 ml = s_ml[(rg * QB + qb) * 64 + lane];
      const float M = fmaxf(m_ref[qb], ml.x);
      const float a0 = m_ref[qb] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m_ref[qb] - M);
      const float a1 = ml.x == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(ml.x - M);
#pragma unroll
      for (int db = 0; db < NDB; ++db)
#pragma unroll
        for (int v = 0; v < 16; ++v)
          o[db][qb][v] = o[db][qb][v] * a0 + xo[(((rg * QB + qb) * NDB + db) * 16 + v) * 64 + lane] * a1;
      lsum[qb] = lsum[qb] * a0 + ml.y * a1;
      m_ref[qb] = M;
    }
  }

  // ---- write this split's unnormalised partial output, reference max and sum
  const size_t obase = ((size_t)bg * splits + split) * mrows_pad;
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    const int qr = row0 + rg * 32 * QB + qb * 32 + l32;
    float* op = wsO + (obase + qr) * HD;
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int r4 = 0; r4 < 4; ++r4) {
        const int d = db * 32 + 8 * r4 + 4 * hl;
        *(float4*)(op + d) = make_float4(o[db][qb][4 * r4], o[db][qb][4 * r4 + 1],
                                         o[db][qb][4 * r4 + 2], o[db][qb][4 * r4 + 3]);
      }
    if (hl == 0) wsML[obase + qr] = make_float2(m_ref[qb], lsum[qb]);
  }
}

template <int HD>
__global__ __launch_bounds__(kThreads) void attn_combine_kernel(
    const float* __restrict__ wsO, const float2* __restrict__ wsML,
    const int32_t* __restrict__ ctxp, const int32_t* __restrict__ nnp, int B, int N, int Hq,
    int Hkv, int max_ctx, int split_len, int splits, int mrows_pad, uint16_t* __restrict__ O) {
  constexpr int TPR = HD / 4;  // threads per output row, 4 values each
  constexpr int RPB = kThreads / TPR;
  const int row = blockIdx.x * RPB + threadIdx.x / TPR;
  const int d = (threadIdx.x % TPR) * 4;
  if (row >= B * N * Hq) return;
  const int hq = row % Hq, i = (row / Hq) % N, b = row / (Hq * N);
  const int n = min(max(nnp[b], 0), N);
  if (i >= n) return;
  const int ctx = min(max(ctxp[b], 0), max_ctx);
  const int R = ctx + n;
  const int G = Hq / Hkv, g = hq / G;
  const int qr = i * G + (hq - g * G);
  const int nspl = (R + split_len - 1) / split_len;
  const size_t base = (size_t)(b * Hkv + g) * splits;
  // loads are issued eight splits at a time so their latencies overlap
  float M = -INFINITY;
  for (int s0 = 0; s0 < nspl; s0 += 8) {
    float mv[8];
#pragma unroll
    for (int t = 0; t < 8; ++t)
      mv[t] = s0 + t < nspl ? wsML[(base + s0 + t) * mrows_pad + qr].x : -INFINITY;
#pragma unroll
    for (int t = 0; t < 8; ++t) M = fmaxf(M, mv[t]);
  }
  float L = 0.f;
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int s0 = 0; s0 < nspl; s0 += 8) {
    float2 ml[8];
    float4 ov[8];
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      const bool ok = s0 + t < nspl;
      ml[t] = ok ? wsML[(base + s0 + t) * mrows_pad + qr] : make_float2(-INFINITY, 0.f);
      ov[t] = ok ? *(const float4*)(wsO + ((base + s0 + t) * mrows_pad + qr) * HD + d)
                 : make_float4(0.f, 0.f, 0.f, 0.f);
    }
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      const float w = ml[t].x == -INFINITY ? 0.f : exp2f(ml[t].x - M);
      L += w * ml[t].y;
      acc.x += w * ov[t].x; acc.y += w * ov[t].y; acc.z += w * ov[t].z; acc.w += w * ov[t].w;
    }
  }
  const float inv = 1.f / L;
  __bf16 r0 = (__bf16)(acc.x * inv), r1 = (__bf16)(acc.y * inv), r2 = (__bf16)(acc.z * inv),
         r3 = (__bf16)(acc.w * inv);
  uint2 pk;
  pk.x = (uint32_t)__builtin_bit_cast(uint16_t, r0) | ((uint32_t)__builtin_bit_cast(uint16_t, r1) << 16);
  pk.y = (uint32_t)__builtin_bit_cast(uint16_t, r2) | ((uint32_t)__builtin_bit_cast(uint16_t, r3) << 16);
  *(uint2*)(O + (((size_t)b * N + i) * Hq + hq) * HD + d) = pk;
}

// ---------------------------------------------------------------- fp32 VALU path
template <int HD>
__global__ __launch_bounds__(kThreads) void attn_f32_kernel(
    const float* __restrict__ Q, const float* __restrict__ Kc, const float* __restrict__ Vc,
    const int64_t* __restrict__ offp, const int32_t* __restrict__ ctxp,
    const int32_t* __restrict__ parentp, const int32_t* __restrict__ nnp, int N, int Hq,
    int Hkv, int max_ctx, float scale, float* __restrict__ O) {
  constexpr int GROUPS = kThreads / HD;  // key groups for the P.V accumulation
  __shared__ float s_q[HD];
  __shared__ float s_p[kThreads];
  __shared__ float s_red[kThreads / 64];
  __shared__ uint64_t s_anc[4];
  __shared__ float s_acc[GROUPS][HD];
  const int i = blockIdx.x, hq = blockIdx.y, b = blockIdx.z;
  const int tid = threadIdx.x;
  const int n = min(max(nnp[b], 0), N);
  if (i >= n) return;
  const int ctx = min(max(ctxp[b], 0), max_ctx);
  const int R = ctx + n;
  const int G = Hq / Hkv, g = hq / G;
  const int64_t kv0 = offp[b];
  const size_t rs = (size_t)Hkv * HD;
  if (tid < HD) s_q[tid] = Q[(((size_t)b * N + i) * Hq + hq) * HD + tid];
  if (tid == 0) {
    uint64_t a[4];
    const int32_t* pp = parentp + (size_t)b * N;
    ancestor_mask(i, [&](int j) { return pp[j]; }, a);
    for (int w = 0; w < 4; ++w) s_anc[w] = a[w];
  }
  __syncthreads();
  float m_run = -INFINITY, l_run = 0.f, acc = 0.f;
  const int dd = tid % HD, grp = tid / HD;
  for (int k0 = 0; k0 < R; k0 += kThreads) {
    const int key = k0 + tid;
    float sc = -INFINITY;
    bool ok = key < R;
    if (ok && key >= ctx) {
      const int t = key - ctx;
      ok = (s_anc[(t >> 6) & 3] >> (t & 63)) & 1ull;
    }
    if (ok) {
      const float* kr = Kc + (size_t)(kv0 + key) * rs + (size_t)g * HD;
      float dot = 0.f;
      for (int d = 0; d < HD; ++d) dot += s_q[d] * kr[d];
      sc = dot * scale;
    }
    // tile max
    float mx = sc;
    for (int off = 32; off >= 1; off >>= 1) mx = fmaxf(mx, __shfl_xor(mx, off));
    if ((tid & 63) == 0) s_red[tid >> 6] = mx;
    __syncthreads();
    mx = s_red[0];
    for (int w = 1; w < kThreads / 64; ++w) mx = fmaxf(mx, s_red[w]);
    __syncthreads();
    const float m_new = fmaxf(m_run, mx);
    const float ref = m_new == -INFINITY ? 0.f : m_new;
    const float pv = ok ? expf(sc - ref) : 0.f;
    s_p[tid] = pv;
    float sum = pv;
    for (int off = 32; off >= 1; off >>= 1) sum += __shfl_xor(sum, off);
    if ((tid & 63) == 0) s_red[tid >> 6] = sum;
    __syncthreads();
    sum = 0.f;
    for (int w = 0; w < kThreads / 64; ++w) sum += s_red[w];
    const float alpha = expf(m_run - ref);
    l_run = l_run * alpha + sum;
    acc *= alpha;
    m_run = m_new;
    for (int j = grp; j < kThreads && k0 + j < R; j += GROUPS) {
      const float pj = s_p[j];
      if (pj != 0.f) acc += pj * Vc[(size_t)(kv0 + k0 + j) * rs + (size_t)g * HD + dd];
    }
    __syncthreads();
  }
  s_acc[grp][dd] = acc;
  __syncthreads();
  if (tid < HD) {
    float t = 0.f;
    for (int gi = 0; gi < GROUPS; ++gi) t += s_acc[gi][tid];
    O[(((size_t)b * N + i) * Hq + hq) * HD + tid] = t / l_run;
  }
}

}  // namespace

AttnPlan plan_attn(int batch, int budget, int Hq, int Hkv, int head_dim, int max_ctx) {
  AttnPlan p;
  const int G = Hq / Hkv;
  const int mrows = budget * G;
  // two waves per SIMD (32 query rows each, two key groups) by default; TAPS_ATTN_PLAN=
  // "qb,wk" selects another instantiation (qb in {1,2}, wk in {1,2}) for tuning
  p.qb = 1;
  p.wk = 2;
  if (const char* e = getenv("TAPS_ATTN_PLAN")) {
    int qb = 0, wk = 0;
    if (sscanf(e, "%d,%d", &qb, &wk) == 2 && (qb == 1 || qb == 2) && (wk == 1 || wk == 2) &&
        !(qb == 2 && wk == 2)) {
      p.qb = qb;
      p.wk = wk;
    }
  }
  p.mtile = 4 * 32 * p.qb;
  p.mtiles = (mrows + p.mtile - 1) / p.mtile;
  // split the keys so that about 256 workgroups run, each with >= 2 iterations
  const int keys = max_ctx + budget;
  const int step = kKT * p.wk;
  const long long base = (long long)batch * Hkv * p.mtiles;
  const int splits = (int)((256 + base - 1) / base);
  int len = (keys + splits - 1) / splits;
  len = ((len + step - 1) / step) * step;
  if (len < 2 * step) len = 2 * step;
  p.split_len = len;
  p.splits = (keys + len - 1) / len;
  (void)head_dim;
  return p;
}

size_t attn_ws_bytes(const AttnPlan& pl, int batch, int /*budget*/, int /*Hq*/, int Hkv,
                     int head_dim) {
  const size_t rows = (size_t)batch * Hkv * pl.splits * (size_t)pl.mtiles * pl.mtile;
  return rows * head_dim * sizeof(float) + rows * sizeof(float2) + 256;
}

hipError_t launch_attn_bf16(const void* Q, const void* K, const void* V, const int64_t* off,
                            const int32_t* ctx, const int32_t* parent, const int32_t* n,
                            int batch, int budget, int Hq, int Hkv, int head_dim, int max_ctx,
                            float scale, const AttnPlan& pl, void* O, void* ws, hipStream_t s,
                            hipEvent_t ev_begin, hipEvent_t ev_end) {
  if (batch <= 0) return hipSuccess;
  const int mrows_pad = pl.mtiles * pl.mtile;
  const size_t rows = (size_t)batch * Hkv * pl.splits * mrows_pad;
  float* wsO = (float*)ws;
  float2* wsML = (float2*)((char*)ws + rows * head_dim * sizeof(float));
  const int pairs = pl.splits * batch * Hkv;
  dim3 grid((unsigned)(8 * pl.mtiles * ((pairs + 7) / 8)));
  dim3 block((unsigned)(256 * pl.wk));
  const float sl2 = scale * kLog2e;
  const uint16_t *q = (const uint16_t*)Q, *k = (const uint16_t*)K, *v = (const uint16_t*)V;
  if (ev_begin && hipEventRecord(ev_begin, s) != hipSuccess) return hipErrorInvalidValue;
#define TAPS_ATT(QB, WK, HD)                                                                  \
  attn_bf16_kernel<QB, WK, HD><<<grid, block, 0, s>>>(q, k, v, off, ctx, parent, n, budget,   \
                                                      Hq, Hkv, max_ctx, sl2, pl.split_len,    \
                                                      pl.splits, pl.mtiles, pairs, mrows_pad, \
                                                      wsO, wsML)
  if (head_dim == 128) {
    if (pl.qb == 2) TAPS_ATT(2, 1, 128);
    else if (pl.wk == 2) TAPS_ATT(1, 2, 128);
    else TAPS_ATT(1, 1, 128);
  } else {
    if (pl.qb == 2) TAPS_ATT(2, 1, 64);
    else if (pl.wk == 2) TAPS_ATT(1, 2, 64);
    else TAPS_ATT(1, 1, 64);
  }
#undef TAPS_ATT
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (ev_end && hipEventRecord(ev_end, s) != hipSuccess) return hipErrorInvalidValue;
  const int rows_out = batch * budget * Hq;
  if (head_dim == 128) {
    const int rpb = kThreads / 32;
    attn_combine_kernel<128><<<dim3((unsigned)((rows_out + rpb - 1) / rpb)), dim3(kThreads), 0, s>>>(
        wsO, wsML, ctx, n, batch, budget, Hq, Hkv, max_ctx, pl.split_len, pl.splits, mrows_pad,
        (uint16_t*)O);
  } else {
    const int rpb = kThreads / 16;
    attn_combine_kernel<64><<<dim3((unsigned)((rows_out + rpb - 1) / rpb)), dim3(kThreads), 0, s>>>(
        wsO, wsML, ctx, n, batch, budget, Hq, Hkv, max_ctx, pl.split_len, pl.splits, mrows_pad,
        (uint16_t*)O);
  }
  return hipGetLastError();
}

hipError_t launch_attn_f32(const float* Q, const float* K, const float* V, const int64_t* off,
                           const int32_t* ctx, const int32_t* parent, const int32_t* n,
                           int batch, int budget, int Hq, int Hkv, int head_dim, int max_ctx,
                           float scale, float* O, hipStream_t s, hipEvent_t ev_begin,
                           hipEvent_t ev_end) {
  if (batch <= 0) return hipSuccess;
  dim3 grid((unsigned)budget, (unsigned)Hq, (unsigned)batch), block(kThreads);
  if (ev_begin && hipEventRecord(ev_begin, s) != hipSuccess) return hipErrorInvalidValue;
  if (head_dim == 128)
    attn_f32_kernel<128><<<grid, block, 0, s>>>(Q, K, V, off, ctx, parent, n, budget, Hq, Hkv, max_ctx, scale, O);
  else
    attn_f32_kernel<64><<<grid, block, 0, s>>>(Q, K, V, off, ctx, parent, n, budget, Hq, Hkv, max_ctx, scale, O);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (ev_end && hipEventRecord(ev_end, s) != hipSuccess) return hipErrorInvalidValue;
  return hipSuccess;
}

}  // namespace taps
