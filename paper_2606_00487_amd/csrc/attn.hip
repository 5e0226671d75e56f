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
#include <algorithm>
#include <cstdio>
#include <cstdlib>
#include <type_traits>

#include <hip/hip_ext.h>

#include "common.h"
#include "ldsload.h"

namespace taps {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

constexpr int kThreads = 256;
constexpr int kWavesA = 4;
constexpr int kKT = 64;  // keys per tile
constexpr float kLog2e = 1.4426950408889634f;


constexpr int kAncWords = TAPS_MAX_BUDGET / 64;   // 64-bit words of one node's mask

// ancestor-or-self mask of node i from parent pointers (a parent outside [0, node) ends
// the walk), kAncWords words in registers; par(j) reads the parent of node j
template <typename F>
__device__ inline void ancestor_mask(int i, F par, uint64_t (&a)[kAncWords]) {
#pragma unroll
  for (int w = 0; w < kAncWords; ++w) a[w] = 0ull;
  int cur = i;
  for (;;) {
    const uint64_t bit = 1ull << (cur & 63);
    const int cw = cur >> 6;
#pragma unroll
    for (int w = 0; w < kAncWords; ++w) a[w] |= cw == w ? bit : 0ull;
    const int p = par(cur);
    if (p < 0 || p >= cur) break;
    cur = p;
  }
}

// 64 tree rows of a node's ancestor-or-self mask (kAncWords words in LDS), starting at
// row t0 (t0 may be negative: rows below 0 read as 0)
__device__ inline uint64_t mask_window(const uint64_t* anc, int t0) {
  if (t0 <= -64 || t0 >= 64 * kAncWords) return 0ull;
  if (t0 < 0) return anc[0] << (-t0);
  const int w = t0 >> 6, sh = t0 & 63;
  const uint64_t lo = anc[w];
  const uint64_t hi = w + 1 < kAncWords ? anc[w + 1] : 0ull;
  return sh ? (lo >> sh) | (hi << (64 - sh)) : lo;
}

// bits j of a 64-bit window for j < 64 (0 for j <= 0, all ones for j >= 64)
__device__ inline uint64_t low_bits(int j) {
  return j <= 0 ? 0ull : (j >= 64 ? ~0ull : ((1ull << j) - 1ull));
}

// four floats rounded to bf16 (nearest even), packed little-endian
__device__ inline uint2 pack_bf16x4(float a, float b, float c, float d) {
  const __bf16 r0 = (__bf16)a, r1 = (__bf16)b, r2 = (__bf16)c, r3 = (__bf16)d;
  uint2 pk;
  pk.x = (uint32_t)__builtin_bit_cast(uint16_t, r0) | ((uint32_t)__builtin_bit_cast(uint16_t, r1) << 16);
  pk.y = (uint32_t)__builtin_bit_cast(uint16_t, r2) | ((uint32_t)__builtin_bit_cast(uint16_t, r3) << 16);
  return pk;
}

// the value held by lane l ^ 32 (a VALU lane swap, no LDS round trip)
__device__ inline float other_half(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                  false);
  // r[0]: lanes 0-31 keep x, lanes 32-63 get x[l-32]; r[1]: lanes 0-31 get x[l+32]
  return __uint_as_float((threadIdx.x & 32) ? r[0] : r[1]);
}

typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;
typedef __attribute__((address_space(3))) void lds_void;

// permutation of all four bits of a row's 16-byte chunk index (the 16 rows a 16-byte
// per-lane read touches at once land on distinct chunk positions, i.e. on all 64 banks)
__device__ inline int kswz16(int r) { return ((r & 3) << 2) | ((r >> 2) & 3); }

typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;

// permutation of a key row's low three bits that XORs its 16-byte chunks: the 8 rows a
// K read touches at once, and the 4 rows x 2 chunk pairs a transposing V read touches
// at once, land on distinct LDS banks
__device__ inline int kswz(int r) { return ((r & 3) << 1) | ((r >> 2) & 1); }

// One workgroup: four waves, 32 query rows each (S^T and O^T tiles of one 32x32 MFMA
// block per 32 keys and per 32 head dimensions), one 64-key stage of K and V per step.
// K and V tiles go from global memory straight into LDS with buffer loads (16 bytes per
// lane), row-major with the 16-byte chunks of key row r XOR-permuted by kswz(r).  The
// buffer resources cover exactly this split's rows, so rows past the split's end read as
// zeros without touching memory: the look-ahead needs no bounds logic.  V^T operands are
// read with the transposing LDS read: in each 16-lane group, lane i gets element i % 4 of
// the 8 bytes read by lanes 4t + i/4 (t = 0..3), i.e. 4 consecutive keys at its d.
//
// Software pipeline over stages i = 0, 1, ...: step i applies the softmax to S(i) and
// accumulates P(i) V(i) while the MFMAs of S(i+1) = K(i+1) Q^T run in between; the loads
// of V(i+3) and K(i+4) are issued at the start of step i, so every load has three steps
// to arrive.  K and V each cycle through NBUF = 4 LDS buffers.
//
// The grid is one-dimensional: the query-row tiles of one (request, KV head, split) get
// block ids that differ by multiples of 8, so they run on the same XCD and share its L2.
template <int HD>
__global__ __launch_bounds__(256) void attn_bf16_w4_kernel(
    const uint16_t* __restrict__ Q, const uint16_t* __restrict__ Kc,
    const uint16_t* __restrict__ Vc, const int64_t* __restrict__ offp,
    const int32_t* __restrict__ ctxp, const int32_t* __restrict__ parentp,
    const int32_t* __restrict__ nnp, int N, int Hq, int Hkv, int max_ctx, float scale_log2,
    int split_len, int splits, int mtiles, int pairs, int mrows_pad, uint16_t* __restrict__ wsO,
    float2* __restrict__ wsML) {
  // the body uses the buffer-resource type, which exists only in the device pass; the
  // host pass needs no more than the signature to emit the launch stub
#if defined(__HIP_DEVICE_COMPILE__)
  constexpr int NT = 256;
  constexpr int NW = 4;
  constexpr int ROWB = HD * 2;        // bytes per K/V row
  constexpr int MT = 4 * 32;          // query rows per workgroup
  constexpr int NDB = HD / 32;        // 32-row blocks of O^T
  constexpr int NKK = HD / 16;        // MFMA k-steps over head_dim
  constexpr int TILEB = kKT * ROWB;   // bytes of one K (or V) tile
  constexpr int BLK = kWave * 16;     // bytes one wave writes per direct load
  constexpr int LPH = TILEB / BLK / NW;  // direct loads per wave per tile
  constexpr int RB = BLK / ROWB;      // key rows per direct load
  constexpr int STEP = kKT;           // keys per stage
  static_assert(TILEB % (BLK * NW) == 0 && LPH >= 1 && 7 * LPH <= 63, "direct loads per wave");
  static_assert(BLK % ROWB == 0, "a direct load covers whole rows");
  constexpr int PPT = (TAPS_MAX_BUDGET + NT - 1) / NT;   // parent pointers per thread
  // separate LDS objects, and every access names its buffer statically: the compiler can
  // then tell that reads of one buffer do not overlap the loads in flight into another
  __shared__ __attribute__((aligned(16))) unsigned char s_k0[TILEB];
  __shared__ __attribute__((aligned(16))) unsigned char s_k1[TILEB];
  __shared__ __attribute__((aligned(16))) unsigned char s_k2[TILEB];
  __shared__ __attribute__((aligned(16))) unsigned char s_k3[TILEB];
  __shared__ __attribute__((aligned(16))) unsigned char s_v0[TILEB];
  __shared__ __attribute__((aligned(16))) unsigned char s_v1[TILEB];
  __shared__ __attribute__((aligned(16))) unsigned char s_v2[TILEB];
  __shared__ __attribute__((aligned(16))) unsigned char s_v3[TILEB];
  __shared__ uint64_t s_anc[MT + 1][kAncWords];   // masks of this tile's nodes
  __shared__ int s_par[TAPS_MAX_BUDGET];

  // ---- which (request, KV head, split, row tile) this workgroup owns
  const int xcd = blockIdx.x & 7, slot = blockIdx.x >> 3;
  const int mt = slot % mtiles, pair = (slot / mtiles) * 8 + xcd;
  if (pair >= pairs) return;
  const int split = pair % splits, bg = pair / splits;
  const int b = bg / Hkv, g = bg - (bg / Hkv) * Hkv;
  const int G = Hq / Hkv;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int rg = wave;
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
  const uint32_t rsb = (uint32_t)(row_stride * 2);   // bytes between consecutive cache rows
  const int nst = (k_end - k_begin + STEP - 1) / STEP;   // stages of this split (>= 1)
  // buffer resources over this split's K and V rows of head g (the host keeps
  // (split_len + 5 * STEP) * rsb below 2^31)
  const size_t seg = ((size_t)kv0 + k_begin) * row_stride + (size_t)g * HD;
  const __amdgpu_buffer_rsrc_t krs = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(Kc + seg), (short)0, (int)((uint32_t)(k_end - k_begin) * rsb), 0x00020000);
  const __amdgpu_buffer_rsrc_t vrs = __builtin_amdgcn_make_buffer_rsrc(
      (void*)(Vc + seg), (short)0, (int)((uint32_t)(k_end - k_begin) * rsb), 0x00020000);

  // ---- direct loads.  Wave w fills blocks w*LPH .. w*LPH + LPH - 1 of a tile; a block is
  // RB whole key rows.  The wave index is made explicitly uniform so that the LDS
  // destinations stay scalar.
  const int wave_u = __builtin_amdgcn_readfirstlane(wave);
  uint32_t ld_off[LPH];    // byte offset of this lane's piece from the stage's first row
#pragma unroll
  for (int j = 0; j < LPH; ++j) {
    const int rb = (wave_u * LPH + j) * BLK + lane * 16;   // byte within the tile
    const int kr = rb / ROWB;
    const int pc = (rb - kr * ROWB) / 16;
    ld_off[j] = (uint32_t)kr * rsb + (uint32_t)((pc ^ kswz(kr)) * 16);
  }
  // stage s of K (or V) into buffer buf; rows past the split's end arrive as zeros (the
  // whole offset goes into the per-lane offset, which the buffer range check covers)
  auto issue = [&](__amdgpu_buffer_rsrc_t rs, unsigned char* buf, int s) __attribute__((always_inline)) {
    const uint32_t soff = (uint32_t)(s * STEP) * rsb;
    unsigned char* dst = buf + wave_u * LPH * BLK;
#pragma unroll
    for (int j = 0; j < LPH; ++j)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_void*)(dst + j * BLK), 16,
                                               ld_off[j] + soff, 0, 0, 0);
  };

  // ---- queries of this lane (B operand of S^T = K Q^T)
  bf16x8 q[NKK];
  int qnode;
  {
    int qr = row0 + rg * 32 + l32;
    qr = min(qr, N * G - 1);
    const int node = qr / G, hq = g * G + (qr - node * G);
    qnode = node;
    const uint16_t* qp = Q + (((size_t)b * N + node) * Hq + hq) * HD;
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk) q[kk] = *(const bf16x8*)(qp + kk * 16 + hl * 8);
  }
  // parent pointers for the ancestor masks
  const bool tree_split = k_end > ctx;
  int my_par[PPT];
#pragma unroll
  for (int j = 0; j < PPT; ++j) {
    const int i = tid + j * NT;
    my_par[j] = tree_split && i < n ? parentp[(size_t)b * N + i] : -1;
  }
  // the tile's nodes: query rows row0 .. row0 + MT - 1 belong to nodes node0 .. node0 + MT
  const int node0 = row0 / G;
  const int node_end = min(n, (row0 + MT - 1) / G + 1);
  // the first stages load while the masks are set up; the queries and parents were
  // issued first, so waiting for them leaves these loads in flight.  The order K(0),
  // [V(0) K(1)], [V(1) K(2)], [V(2) K(3)] matches the steps' [V(i+3) K(i+4)].
  issue(krs, s_k0, 0);
  issue(vrs, s_v0, 0);
  issue(krs, s_k1, 1);
  issue(vrs, s_v1, 1);
  issue(krs, s_k2, 2);
  issue(vrs, s_v2, 2);
  issue(krs, s_k3, 3);
  TAPS_WAIT_VMCNT(7 * LPH);

  // ---- ancestor-or-self masks of the tree rows, in LDS (read only by masked tiles)
  if (tree_split) {
#pragma unroll
    for (int j = 0; j < PPT; ++j)
      if (tid + j * NT < n) s_par[tid + j * NT] = my_par[j];
    __syncthreads();
    for (int i = node0 + tid; i < node_end; i += NT) {
      uint64_t a[kAncWords];
      ancestor_mask(i, [&](int j) { return s_par[j]; }, a);
#pragma unroll
      for (int w = 0; w < kAncWords; ++w) s_anc[i - node0][w] = a[w];
    }
    __syncthreads();
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

  // S^T of 32-key block kb of the tile in K buffer kbuf, one k-step
  auto s_mfma = [&](const unsigned char* kbuf, int kb, int kk, f32x16 (&s)[2])
      __attribute__((always_inline)) {
    const bf16x8 a = *(const bf16x8*)(kbuf + kb * 32 * ROWB + 32 * (kk & ~3) + koff[kk & 3]);
    if (kk == 0) {
      f32x16 z;
#pragma unroll
      for (int v = 0; v < 16; ++v) z[v] = 0.f;
      s[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, q[kk], z, 0, 0, 0);
    } else {
      s[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, q[kk], s[kb], 0, 0, 0);
    }
  };

  f32x16 o[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db)
#pragma unroll
    for (int v = 0; v < 16; ++v) o[db][v] = 0.f;
  float m_ref = -INFINITY, l_run = 0.f;

  // Softmax of S(i) (keys base ...) and O^T += V(i)^T P(i)^T from V buffer vbuf, with
  // the MFMAs of S(i+1) from K buffer knext interleaved
  auto softmax_pv = [&](f32x16 (&sc)[2], const unsigned char* vbuf, const unsigned char* knext,
                        f32x16 (&sn)[2], int base) __attribute__((always_inline)) {
    // ---- mask (only tiles that reach the tree rows or the split end)
    const bool need_mask = base + kKT > ctx || base + kKT > k_end;
    if (need_mask) {
      const uint64_t win =
          base + kKT > ctx && qnode < n ? mask_window(s_anc[qnode - node0], base - ctx) : 0ull;
      uint64_t A = (low_bits(ctx - base) | win) & low_bits(k_end - base);
      A >>= 4 * hl;   // this lane's keys are kb*32 + 8*(v/4) + 4*hl + v%4
      const uint32_t mlo = (uint32_t)A, mhi = (uint32_t)(A >> 32);
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const uint32_t word = kb ? mhi : mlo;
          const bool ok = (word >> (8 * (v >> 2) + (v & 3))) & 1u;
          sc[kb][v] = ok ? sc[kb][v] : -INFINITY;
        }
    }
    // ---- first key block of S(i+1) while the row maximum of S(i) is found
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk) s_mfma(knext, 0, kk, sn);
    float mx = -INFINITY;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int v = 0; v < 16; ++v) mx = fmaxf(mx, sc[kb][v]);
    mx = fmaxf(mx, other_half(mx)) * scale_log2;   // scale > 0
    // move the reference max only when it is exceeded by more than 2^8
    const bool upd = mx > m_ref + 8.f;
    if (__ballot(upd)) {
      const float nref = upd ? mx : m_ref;
      const float alpha = upd ? __builtin_amdgcn_exp2f(m_ref - nref) : 1.f;
      l_run *= alpha;
#pragma unroll
      for (int db = 0; db < NDB; ++db)
#pragma unroll
        for (int v = 0; v < 16; ++v) o[db][v] *= alpha;
      m_ref = nref;
    }
    const float nref = m_ref == -INFINITY ? 0.f : -m_ref;
    // ---- P = exp2(scale*s - ref) and O^T += V^T P^T in four groups of 8 keys per lane
    // half; the second key block of S(i+1) goes into groups 2 and 3, after the first key
    // block of S(i) is dead
#pragma unroll
    for (int grp = 0; grp < 4; ++grp) {
      const int kb = grp >> 1, hf = grp & 1;
      bf16x8 pg;
      float sum = 0.f;
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        const float e = __builtin_amdgcn_exp2f(fmaf(sc[kb][hf * 8 + t], scale_log2, nref));
        sum += e;
        pg[t] = (__bf16)e;
      }
      l_run += sum;
#pragma unroll
      for (int db = 0; db < NDB; ++db) {
        const unsigned char* va = vbuf + voff[db & 1] + ((kb * 32 + 16 * hf) * ROWB + 64 * (db & ~1));
        const unsigned char* vb = vbuf + voff[db & 1] + ((kb * 32 + 16 * hf + 8) * ROWB + 64 * (db & ~1));
        const bf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)va);
        const bf16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)vb);
        const bf16x8 a = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
        o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pg, o[db], 0, 0, 0);
      }
      if (grp >= 2) {
#pragma unroll
        for (int kk = (grp - 2) * (NKK / 2); kk < (grp - 1) * (NKK / 2); ++kk) s_mfma(knext, 1, kk, sn);
      }
    }
  };

  // step i: V(i+3) and K(i+4) start loading, then the softmax and P V of stage i run
  // together with S(i+1).  Buffers: K(i+4) replaces K(i), V(i+3) replaces V(i-1).
  auto step = [&](f32x16 (&sc)[2], f32x16 (&sn)[2], unsigned char* k_free,
                  const unsigned char* k_next, const unsigned char* v_cur, unsigned char* v_free,
                  int i) __attribute__((always_inline)) {
    issue(vrs, v_free, i + 3);
    issue(krs, k_free, i + 4);
    TAPS_WAIT_VMCNT(6 * LPH);         // V(i) and K(i+1) have landed (this wave's part)
    TAPS_STAGE_BARRIER();             // ... and every other wave's part
    softmax_pv(sc, v_cur, k_next, sn, k_begin + i * STEP);
    TAPS_STAGE_BARRIER();             // the buffers of K(i+1) and V(i) may be refilled
  };

  // ---- S(0), then the steps, unrolled by four so that every access names its buffer
  f32x16 sA[2], sB[2];
  TAPS_WAIT_VMCNT(6 * LPH);           // K(0)
  TAPS_STAGE_BARRIER();
#pragma unroll
  for (int kb = 0; kb < 2; ++kb)
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk) s_mfma(s_k0, kb, kk, sA);
  for (int i = 0;;) {
    step(sA, sB, s_k0, s_k1, s_v0, s_v3, i);
    if (++i >= nst) break;
    step(sB, sA, s_k1, s_k2, s_v1, s_v0, i);
    if (++i >= nst) break;
    step(sA, sB, s_k2, s_k3, s_v2, s_v1, i);
    if (++i >= nst) break;
    step(sB, sA, s_k3, s_k0, s_v3, s_v2, i);
    if (++i >= nst) break;
  }
  // the look-ahead loads past the split's end read nothing from memory; let them land
  // before the workgroup's LDS is released
  TAPS_WAIT_VMCNT(0);

  const float lsum = l_run + other_half(l_run);
  const float inv = lsum > 0.f ? 1.f / lsum : 0.f;

  // ---- write this split's partial: O / sum in bf16, reference max and sum
  const size_t obase = ((size_t)bg * splits + split) * mrows_pad;
  const int qr = row0 + rg * 32 + l32;
  uint16_t* op = wsO + (obase + qr) * HD;
#pragma unroll
  for (int db = 0; db < NDB; ++db)
#pragma unroll
    for (int r4 = 0; r4 < 4; ++r4) {
      const int d = db * 32 + 8 * r4 + 4 * hl;
      *(uint2*)(op + d) = pack_bf16x4(o[db][4 * r4] * inv, o[db][4 * r4 + 1] * inv,
                                      o[db][4 * r4 + 2] * inv, o[db][4 * r4 + 3] * inv);
    }
  if (hl == 0) wsML[obase + qr] = make_float2(m_ref, lsum);
#endif
}

// Eight waves per workgroup (two per SIMD), in two key groups of four: group g works on
// the 32-key stages g, g + 2, g + 4, ... of the split, each wave on 32 query rows, and
// the groups merge their results through LDS at the end.  K and V cycle through rings of
// eight 32-key slots (sixteen separate LDS objects): step t processes stages 2t and
// 2t + 1 and issues the loads of V(2t + 6), V(2t + 7), K(2t + 8) and K(2t + 9), so every
// load has three steps to arrive.  Within a group the pipeline is the same as in the
// four-wave kernel: the softmax and P V of a stage run together with the MFMAs of S for
// the group's next stage.  The step loop is written once per group (template) and
// unrolled by four, so that every LDS access names its slot statically.
// Division of small non-negative ints by the launch's tile, split, head and group
// counts: floor(n / d) = high half of n * ceil(2^32 / d), exact for n < 2^32 / d (the
// rounding term of the multiplier adds less than n / 2^32 < 1/d to n / d)
struct DivMagic {
  uint32_t mt, sp, hk, g;
  __device__ int div(int n, int d, uint32_t m) const {
    return d == 1 ? n : (int)__umulhi((uint32_t)n, m);
  }
  static uint32_t make(int d) {
    return d > 1 ? (uint32_t)((0x100000000ull + (uint64_t)d - 1) / (uint64_t)d) : 0u;
  }
};

// (Paged KV: pages of 32 .. 4096 rows, so a 32-key stage never straddles two pages.)
// page ids of one split held in LDS (they share the (max, sum) exchange buffer, which is
// used only after the key loop); split lengths are capped so that a split spans at most
// this many pages
constexpr int kPageSlots = 1024;

// The request's context length, node count and KV offset in one scalar-memory round
// trip (issued together, then one wait)
__device__ inline void load_request_scalars(const int32_t* c, const int32_t* nn,
                                            const int64_t* o, int& cv, int& nv, int64_t& ov) {
  asm volatile(
      "s_load_dword %0, %3, 0x0\n\t"
      "s_load_dword %1, %4, 0x0\n\t"
      "s_load_dwordx2 %2, %5, 0x0\n\t"
      "s_waitcnt lgkmcnt(0)"
      : "=&s"(cv), "=&s"(nv), "=&s"(ov)
      : "s"(c), "s"(nn), "s"(o)
      : "memory");
}

// the request's context length and node count plus four ints of its block-table row (the
// pages of the split's first four stages) in one scalar-memory round trip
__device__ inline void load_request_pages(const int32_t* c, const int32_t* nn,
                                          const int32_t* p0, const int32_t* p1,
                                          const int32_t* p2, const int32_t* p3, int& cv,
                                          int& nv, int& v0, int& v1, int& v2, int& v3) {
  asm volatile(
      "s_load_dword %0, %6, 0x0\n\t"
      "s_load_dword %1, %7, 0x0\n\t"
      "s_load_dword %2, %8, 0x0\n\t"
      "s_load_dword %3, %9, 0x0\n\t"
      "s_load_dword %4, %10, 0x0\n\t"
      "s_load_dword %5, %11, 0x0\n\t"
      "s_waitcnt lgkmcnt(0)"
      : "=&s"(cv), "=&s"(nv), "=&s"(v0), "=&s"(v1), "=&s"(v2), "=&s"(v3)
      : "s"(c), "s"(nn), "s"(p0), "s"(p1), "s"(p2), "s"(p3)
      : "memory");
}

// two per-request ints in one scalar-memory round trip
__device__ inline void load_two_scalars(const int32_t* x, const int32_t* y, int& xv, int& yv) {
  asm volatile(
      "s_load_dword %0, %2, 0x0\n\t"
      "s_load_dword %1, %3, 0x0\n\t"
      "s_waitcnt lgkmcnt(0)"
      : "=&s"(xv), "=&s"(yv)
      : "s"(x), "s"(y)
      : "memory");
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

// sum of a 64-bit integer over the lanes of a wave, in every lane
__device__ inline long long wave_sum_i64(long long v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) {
    const uint32_t lo = __shfl_xor((uint32_t)v, m), hi = __shfl_xor((uint32_t)((uint64_t)v >> 32), m);
    v += (long long)(((uint64_t)hi << 32) | lo);
  }
  return v;
}

// Ragged work list of several requests.  Request b has R_b keys (context rows + nodes) and
// S_b = ceil(R_b / L) splits per KV head; its pairs are numbered from the prefix sum E_b of
// Hkv * S_b, KV head by KV head.  When the lengths are close (the longest at most 5/4 of
// the mean), L is the host's split length for max_ctx + budget keys, as in the one-request
// plan; otherwise L is sized from the batch's total keys so that the batch makes about
// target_pairs pairs.  Every wave of the workgroup computes the same result; wave 0 of the
// designated workgroup also writes tab[b] = (E_b, S_b) and tab[batch] = (L, total pairs)
// for the split combine.
struct RaggedPick {
  int b, g, split, L;
  bool found;
};
__device__ inline RaggedPick ragged_pick(const int32_t* ctxp, const int32_t* nnp, int batch,
                                         int N, int max_ctx, int Hkv, int target_pairs,
                                         int lcap, int L_host, int p, int2* tab, bool write_tab) {
  const int lane = threadIdx.x & 63;
  long long tot = 0;
  int rmax = 0;
  for (int c = 0; c < batch; c += 64) {
    const int b = c + lane;
    if (b < batch) {
      const int R = min(max(ctxp[b], 0), max_ctx) + min(max(nnp[b], 0), N);
      tot += R;
      rmax = max(rmax, R);
    }
  }
  tot = wave_sum_i64(tot);
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) rmax = max(rmax, __shfl_xor(rmax, m));
  int L;
  if (4ll * rmax * batch <= 5ll * tot) {
    L = L_host;
  } else {
    const long long want = (tot * Hkv + target_pairs - 1) / target_pairs;
    L = (int)min((long long)lcap, max(128ll, (want + 63) / 64 * 64));
  }
  RaggedPick r;
  r.b = r.g = r.split = 0;
  r.L = L;
  r.found = false;
  int carry = 0;
  for (int c = 0; c < batch; c += 64) {
    const int b = c + lane;
    int R = 0;
    if (b < batch) R = min(max(ctxp[b], 0), max_ctx) + min(max(nnp[b], 0), N);
    const int S = (R + L - 1) / L;
    const int P = Hkv * S;
    const int incl = carry + wave_inclusive_sum(P);
    const int excl = incl - P;
    if (write_tab && b < batch) tab[b] = make_int2(excl, S);
    const uint64_t m = __ballot(b < batch && P > 0 && excl <= p && p < incl);
    if (m && !r.found) {
      const int l = __ffsll((long long)m) - 1;
      const int local = p - __builtin_amdgcn_readlane(excl, l);
      const int Sb = __builtin_amdgcn_readlane(S, l);
      r.b = c + l;
      r.g = local / Sb;
      r.split = local - r.g * Sb;
      r.found = true;
    }
    carry = __builtin_amdgcn_readlane(incl, 63);
  }
  if (write_tab && lane == 0) tab[batch] = make_int2(L, carry);
  return r;
}

template <int KG>
struct GroupTag {
  static constexpr int value = KG;
};

// The body of both bf16 kernels below.  PAGED: K and V are page pools
// [num_pages][page_rows][Hkv][HD] and request b's logical row r sits at page
// btab[b][r >> page_shift], slot r & (page_rows - 1) (offp unused); otherwise Kc and Vc are
// the contiguous cache and request b starts at row offp[b].  The body uses the
// buffer-resource type, which exists only in the device pass; the host pass needs no more
// than the kernels' signatures to emit their launch stubs.
#if defined(__HIP_DEVICE_COMPILE__)
template <bool PAGED>
__device__ __attribute__((always_inline)) inline void attn_bf16_body(
    const uint16_t* __restrict__ Q, const uint16_t* __restrict__ Kc,
    const uint16_t* __restrict__ Vc, const int64_t* __restrict__ offp,
    const int32_t* __restrict__ ctxp, const int32_t* __restrict__ parentp,
    const int32_t* __restrict__ nnp, int N, int Hq, int Hkv, int max_ctx, float scale_log2,
    int split_len, int splits, int mtiles, int pairs, int mrows_pad, uint16_t* __restrict__ wsO,
    float2* __restrict__ wsML, DivMagic dm, int batch, int target_pairs, int lcap,
    int2* __restrict__ tab, const PagedKV& pk) {
  constexpr int HD = 128;
  constexpr int NT = 512;
  constexpr int ROWB = HD * 2;        // bytes per K/V row
  constexpr int MT = 4 * 32;          // query rows per workgroup
  constexpr int NDB = HD / 32;        // 32-row blocks of O^T
  constexpr int NKK = HD / 16;        // MFMA k-steps over head_dim
  constexpr int KT = 32;              // keys per stage
  constexpr int TILEB = KT * ROWB;    // 8 KB: one K (or V) slot
  constexpr int BLK = kWave * 16;     // bytes one wave writes per direct load
  static_assert(TILEB == 8 * BLK, "one direct load per wave and slot");
  static_assert(NT >= TAPS_MAX_BUDGET, "one parent pointer per thread");
  static_assert(TAPS_MAX_BUDGET <= 8 * 64, "the eight waves load 64 parent pointers each");
  __shared__ __attribute__((aligned(16))) unsigned char s_k0[TILEB], s_k1[TILEB], s_k2[TILEB],
      s_k3[TILEB], s_k4[TILEB], s_k5[TILEB], s_k6[TILEB], s_k7[TILEB];
  __shared__ __attribute__((aligned(16))) unsigned char s_v0[TILEB], s_v1[TILEB], s_v2[TILEB],
      s_v3[TILEB], s_v4[TILEB], s_v5[TILEB], s_v6[TILEB], s_v7[TILEB];
  __shared__ uint64_t s_anc[MT + 1][kAncWords];   // masks of this tile's nodes
  __shared__ int s_par[TAPS_MAX_BUDGET];
  __shared__ float2 s_ml[8 * 64];

  // every kernel argument into scalar registers at once: one round trip for all of them
  // instead of one per first use
  asm volatile("" ::"s"(Q), "s"(Kc), "s"(Vc), "s"(offp), "s"(ctxp), "s"(parentp), "s"(nnp),
               "s"(N), "s"(Hq), "s"(Hkv), "s"(max_ctx), "s"(scale_log2), "s"(split_len),
               "s"(splits), "s"(mtiles), "s"(pairs), "s"(mrows_pad), "s"(wsO), "s"(wsML),
               "s"(dm.mt), "s"(dm.sp), "s"(dm.hk), "s"(dm.g));
  if constexpr (PAGED)
    asm volatile("" ::"s"(pk.btab), "s"(pk.max_pages), "s"(pk.num_pages), "s"(pk.page_shift));
  // ---- which (request, KV head, split, row tile) this workgroup owns.  The row tiles of a
  // pair are 8 block ids apart (one XCD, which shares the pair's K/V in its L2).  One
  // request (tab == nullptr): pair = (KV head) * splits + split, fixed by the host, and each
  // XCD takes a run of consecutive pairs, so that the splits of a KV head, which all read
  // its query tile, share that tile in one L2; several: the ragged list of ragged_pick, its
  // pairs interleaved over the XCDs (the host sizes the grid for the most pairs there can
  // be).  The split's partial results go to slot `pair`.
  const int xcd = blockIdx.x & 7, slot = blockIdx.x >> 3;
  const int sq = dm.div(slot, mtiles, dm.mt);
  const int mt = slot - sq * mtiles;
  const int pair = tab == nullptr ? xcd * ((pairs + 7) >> 3) + sq : sq * 8 + xcd;
  if (pair >= pairs) return;
  int b, g, split;
  if (tab == nullptr) {
    const int bg = dm.div(pair, splits, dm.sp);
    split = pair - bg * splits;
    b = dm.div(bg, Hkv, dm.hk);
    g = bg - b * Hkv;
  } else {
    const RaggedPick rp = ragged_pick(ctxp, nnp, batch, N, max_ctx, Hkv, target_pairs, lcap,
                                      split_len, pair, tab,
                                      pair == 0 && mt == 0 && (threadIdx.x >> 6) == 0);
    if (!rp.found) return;   // past the batch's pairs (nothing issued yet)
    b = rp.b;
    g = rp.g;
    split = rp.split;
    split_len = rp.L;
  }
  const int G = dm.div(Hq, Hkv, dm.hk);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int rg = wave & 3, kg = wave >> 2;
  const int l32 = lane & 31, hl = lane >> 5;
  const int row0 = mt * MT;

  // ---- the query tile and the parent pointers go straight into LDS first (their
  // addresses do not depend on the request's sizes): V slots 4-7 are free until after
  // the first S.  Every global read of this kernel is such a direct load, issued as inline
  // assembly and ordered by explicit vmcnt waits.  Tile row r (query row row0 + r: node
  // (row0 + r) / G, query head g * G + (row0 + r) % G) is in V slot 4 + r / 32, its 16-byte
  // chunks XOR-permuted by kswz16(r % 32); wave (rg, kg) loads rows rg * 32 + kg * 16 ..
  // + 15, four rows (1 KB) per load.
  const int wave_u = __builtin_amdgcn_readfirstlane(wave);
  const int rg_u = wave_u & 3, kg_u = wave_u >> 2;
  unsigned char* const qslot = rg_u == 0 ? s_v4 : rg_u == 1 ? s_v5 : rg_u == 2 ? s_v6 : s_v7;
  {
    const i32x4 qrs = buffer_rsrc(Q + (size_t)b * N * Hq * HD, (uint32_t)((size_t)N * Hq * HD * 2));
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int r = kg_u * 16 + 4 * j + (lane >> 4);   // row within the slot
      const int qr = min(row0 + rg_u * 32 + r, N * G - 1);
      const int node = dm.div(qr, G, dm.g);
      const uint32_t off = (uint32_t)(node * Hq + g * G + (qr - node * G)) * (HD * 2) +
                           16u * (uint32_t)((lane & 15) ^ kswz16(r));
      load_lds16(qrs, qslot + (kg_u * 16 + 4 * j) * ROWB, off);
    }
    if (wave_u < TAPS_MAX_BUDGET / 64)
      load_lds4(buffer_rsrc(parentp + (size_t)b * N, (uint32_t)N * 4),
                (unsigned char*)s_par + 256 * wave_u, (uint32_t)(64 * wave_u + lane) * 4);
  }
  // paged: the block-table entries of this split's pages (entries past the row read 0)
  int* const s_pg = (int*)s_ml;
  static_assert(sizeof(s_ml) >= kPageSlots * sizeof(int), "page ids fit the exchange buffer");
  int pi0 = 0;
  if constexpr (PAGED) {
    pi0 = (split * split_len) >> pk.page_shift;
    const i32x4 prs = buffer_rsrc(pk.btab + (size_t)b * pk.max_pages, (uint32_t)pk.max_pages * 4);
#pragma unroll
    for (int j = 0; j < kPageSlots / 512; ++j)
      load_lds4(prs, (unsigned char*)s_pg + 256 * (wave_u + 8 * j),
                (uint32_t)(pi0 + 64 * (wave_u + 8 * j) + lane) * 4);
  }
  int qnode;
  {
    const int qr = min(row0 + rg * 32 + l32, N * G - 1);
    qnode = dm.div(qr, G, dm.g);
  }
  // the tile's nodes: query rows row0 .. row0 + MT - 1 belong to nodes node0 .. node0 + MT
  const int node0 = dm.div(row0, G, dm.g);

  int ctx_raw, n_raw;
  int64_t kv0 = 0;
  int fpg[4] = {0, 0, 0, 0};   // paged: the pages of the split's first four stages
  if constexpr (PAGED) {
    // the entries' addresses are uniform; readfirstlane puts them in scalar registers
    auto entry = [&](int j) {
      const uint64_t a = (uint64_t)(pk.btab + (size_t)b * pk.max_pages +
                                    min(pi0 + j, pk.max_pages - 1));
      return (const int32_t*)(((uint64_t)__builtin_amdgcn_readfirstlane((uint32_t)(a >> 32))
                               << 32) |
                              (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)a));
    };
    load_request_pages(ctxp + b, nnp + b, entry(0), entry(1), entry(2), entry(3), ctx_raw,
                       n_raw, fpg[0], fpg[1], fpg[2], fpg[3]);
  } else {
    load_request_scalars(ctxp + b, nnp + b, offp + b, ctx_raw, n_raw, kv0);
  }
  const int ctx = min(max(ctx_raw, 0), max_ctx);
  const int n = min(max(n_raw, 0), N);
  const int R = ctx + n;
  const int k_begin = split * split_len;
  const int k_end = min(R, k_begin + split_len);
  if (k_begin >= k_end || row0 >= n * G) {
    TAPS_WAIT_VMCNT(0);   // the direct loads into LDS land before the LDS is released
    return;
  }
  const size_t row_stride = (size_t)Hkv * HD;
  const uint32_t rsb = (uint32_t)(row_stride * 2);
  const int nst = (k_end - k_begin + KT - 1) / KT;   // 32-key stages of this split
  const int steps = (nst + 1) / 2;                    // each step: one stage per group
  // buffer resources over this split's K and V rows of head g: rows past the split's end
  // read as zeros without touching memory (the host keeps the range below 2^31 bytes)
  // contiguous: one resource per operand over the split's rows; paged: the pool's head-g
  // column, with a resource per stage (issue below)
  // (paged: as 64-bit integers held in scalar registers)
  auto uniform_ptr = [](const uint16_t* p) -> uint64_t {
    const uint64_t a = (uint64_t)p;
    return ((uint64_t)__builtin_amdgcn_readfirstlane((uint32_t)(a >> 32)) << 32) |
           (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)a);
  };
  const auto krs = [&] {
    if constexpr (PAGED) return uniform_ptr(Kc + (size_t)g * HD);
    else return buffer_rsrc(Kc + ((size_t)kv0 + k_begin) * row_stride + (size_t)g * HD,
                            (uint32_t)(k_end - k_begin) * rsb);
  }();
  const auto vrs = [&] {
    if constexpr (PAGED) return uniform_ptr(Vc + (size_t)g * HD);
    else return buffer_rsrc(Vc + ((size_t)kv0 + k_begin) * row_stride + (size_t)g * HD,
                            (uint32_t)(k_end - k_begin) * rsb);
  }();

  // ---- direct loads: wave w fills block w (rows 4w .. 4w + 3) of every slot
  uint32_t ld_off;
  {
    const int rb = wave_u * BLK + lane * 16;
    const int kr = rb / ROWB;
    const int pc = (rb - kr * ROWB) / 16;
    ld_off = (uint32_t)kr * rsb + (uint32_t)((pc ^ kswz(kr)) * 16);
  }
  // paged steps: waves 2q and 2q + 1 load all of the step's q-th stage, blocks 4 (w & 1) ..
  // 4 (w & 1) + 3 each, so that a wave builds one resource per step instead of four
  uint32_t pg_off[4] = {0u, 0u, 0u, 0u};
  if constexpr (PAGED) {
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      const int rb = (4 * (wave_u & 1) + b) * BLK + lane * 16;
      const int kr = rb / ROWB;
      const int pc = (rb - kr * ROWB) / 16;
      pg_off[b] = (uint32_t)kr * rsb + (uint32_t)((pc ^ kswz(kr)) * 16);
    }
  }
  // contiguous: the stage's offset goes into the per-lane offset, which the buffer range
  // check covers.  Paged: a resource over the stage's rows in page pg, cut at the split's end
  // (rows past it, and whole stages past it, read as zeros without touching memory); page
  // ids outside the pool are clamped into it, so no id reads outside the pool.  Everything
  // here is uniform over the workgroup and kept in scalar registers.
  const int kb_u = __builtin_amdgcn_readfirstlane(k_begin);
  const int ke_u = __builtin_amdgcn_readfirstlane(k_end);
  auto issue_at = [&](const auto& src, unsigned char* buf, int s, int pg)
                      __attribute__((always_inline)) {
    if constexpr (!PAGED) {
      load_lds16(src, buf + wave_u * BLK, ld_off + (uint32_t)(s * KT) * rsb);
    } else {
      // a stage with no rows left gets an empty resource and touches no memory, whatever
      // its page; the host keeps num_pages * page_rows below 2^32 (prow fits 32 bits)
      const int r0 = kb_u + s * KT;                 // logical row of the stage's first key
      const int rows = min(max(ke_u - r0, 0), KT);
      const uint32_t prow = ((uint32_t)min(max(pg, 0), pk.num_pages - 1) << pk.page_shift) |
                            (uint32_t)(r0 & ((1 << pk.page_shift) - 1));
      const uint64_t a = src + (uint64_t)prow * rsb;
      i32x4 r;                          // (readfirstlane: the words stay scalar)
      r[0] = __builtin_amdgcn_readfirstlane((int)(uint32_t)a);
      r[1] = __builtin_amdgcn_readfirstlane((int)(uint32_t)(a >> 32));
      r[2] = __builtin_amdgcn_readfirstlane((int)((uint32_t)rows * rsb));
      r[3] = 0x00020000;
      load_lds16(r, buf + wave_u * BLK, ld_off);
    }
  };
  // paged: the page of stage s < 4 (taken with the request's sizes) ...
  auto first_page = [&](int s) -> int {
    const int j = ((kb_u + s * KT) >> pk.page_shift) - pi0;
    return j <= 0 ? fpg[0] : j == 1 ? fpg[1] : j == 2 ? fpg[2] : fpg[3];
  };
  // ... and of the four stages s0 .. s0 + 3, read from the LDS table (the step reads the
  // next step's pages, so their latency is hidden behind its compute)
  auto read_pages4 = [&](int s0, int (&v)[4]) __attribute__((always_inline)) {
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int r0 = kb_u + (s0 + q) * KT;
      v[q] = s_pg[min((r0 >> pk.page_shift) - pi0, kPageSlots - 1)];
    }
  };
  auto issue = [&](const auto& src, unsigned char* buf, int s) __attribute__((always_inline)) {
    issue_at(src, buf, s, PAGED ? first_page(s) : 0);
  };
  auto page_of_stage = [&](int st) -> int {
    return s_pg[min(((kb_u + st * KT) >> pk.page_shift) - pi0, kPageSlots - 1)];
  };
  // paged: this wave's four blocks of stage st (page pg) into slot buf
  auto issue4_paged = [&](uint64_t src, unsigned char* buf, int st, int pg)
                          __attribute__((always_inline)) {
    const int r0 = kb_u + st * KT;
    const int rows = min(max(ke_u - r0, 0), KT);
    const uint32_t prow = ((uint32_t)min(max(pg, 0), pk.num_pages - 1) << pk.page_shift) |
                          (uint32_t)(r0 & ((1 << pk.page_shift) - 1));
    const uint64_t a = src + (uint64_t)prow * rsb;
    i32x4 r;
    r[0] = __builtin_amdgcn_readfirstlane((int)(uint32_t)a);
    r[1] = __builtin_amdgcn_readfirstlane((int)(uint32_t)(a >> 32));
    r[2] = __builtin_amdgcn_readfirstlane((int)((uint32_t)rows * rsb));
    r[3] = 0x00020000;
#pragma unroll
    for (int b = 0; b < 4; ++b)
      load_lds16(r, buf + (4 * (wave_u & 1) + b) * BLK, pg_off[b]);
  };

  const bool tree_split = k_end > ctx;
  // K(0) K(1) and the loads of step -3 [V(2t+6) V(2t+7) K(2t+8) K(2t+9)] now; those of
  // steps -2 and -1 after the first S (so its reads of K(0), K(1) wait for nothing else)
  issue(krs, s_k0, 0);
  issue(krs, s_k1, 1);
  issue(vrs, s_v0, 0); issue(vrs, s_v1, 1); issue(krs, s_k2, 2); issue(krs, s_k3, 3);
  TAPS_WAIT_VMCNT(6);   // queries and parents: this wave's part
  TAPS_LDS_BARRIER();   // ... and every other wave's part (the K/V loads stay in flight)
  bf16x8 q[NKK];        // queries of this lane: B operand of S^T = K Q^T
#pragma unroll
  for (int kk = 0; kk < NKK; ++kk)
    q[kk] = *(const bf16x8*)(qslot + l32 * ROWB + 16 * ((2 * kk + hl) ^ kswz16(l32)));

  // ---- ancestor-or-self masks of the tree rows, in LDS (read only by masked tiles)
  if (tree_split) {
    const int node_end = min(n, dm.div(row0 + MT - 1, G, dm.g) + 1);
    for (int i = node0 + tid; i < node_end; i += NT) {
      uint64_t a[kAncWords];
      ancestor_mask(i, [&](int j) { return s_par[j]; }, a);
#pragma unroll
      for (int w = 0; w < kAncWords; ++w) s_anc[i - node0][w] = a[w];
    }
    TAPS_LDS_BARRIER();
  }

  // ---- per-lane LDS read offsets
  const int fk = kswz(l32);
  int koff[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) koff[j] = l32 * ROWB + 32 * (j ^ (fk >> 1)) + 16 * (hl ^ (fk & 1));
  const int g16 = (lane >> 4) & 1, tq = (lane & 15) >> 2, qq = lane & 3;
  const int fv = kswz(4 * hl + tq);
  int voff[2];
#pragma unroll
  for (int j = 0; j < 2; ++j)
    voff[j] = (4 * hl + tq) * ROWB + 8 * (qq & 1) + 16 * ((g16 * 2 + (qq >> 1)) ^ (fv & 3)) +
              64 * (j ^ (fv >> 2));

  // S^T of the 32 keys in K slot kbuf, one k-step
  auto s_mfma = [&](const unsigned char* kbuf, int kk, f32x16& s) __attribute__((always_inline)) {
    const bf16x8 a = *(const bf16x8*)(kbuf + 32 * (kk & ~3) + koff[kk & 3]);
    if (kk == 0) {
      f32x16 z;
#pragma unroll
      for (int v = 0; v < 16; ++v) z[v] = 0.f;
      s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, q[kk], z, 0, 0, 0);
    } else {
      s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, q[kk], s, 0, 0, 0);
    }
  };

  f32x16 o[NDB];
#pragma unroll
  for (int db = 0; db < NDB; ++db)
#pragma unroll
    for (int v = 0; v < 16; ++v) o[db][v] = 0.f;
  float m_ref = -INFINITY, l_run = 0.f;

  // Softmax of S (keys base .. base + 31) and O^T += V^T P^T from V slot vbuf, with the
  // MFMAs of the group's next S from K slot knext interleaved
  auto softmax_pv = [&](f32x16& sc, const unsigned char* vbuf, const unsigned char* knext,
                        f32x16& sn, int base) __attribute__((always_inline)) {
    const bool need_mask = base + KT > ctx || base + KT > k_end;
    if (need_mask) {
      const uint64_t win =
          base + KT > ctx && qnode < n ? mask_window(s_anc[qnode - node0], base - ctx) : 0ull;
      uint64_t A = (low_bits(ctx - base) | win) & low_bits(k_end - base);
      const uint32_t word = (uint32_t)(A >> (4 * hl));   // keys 8*(v/4) + 4*hl + v%4
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const bool ok = (word >> (8 * (v >> 2) + (v & 3))) & 1u;
        sc[v] = ok ? sc[v] : -INFINITY;
      }
    }
#pragma unroll
    for (int kk = 0; kk < NKK / 2; ++kk) s_mfma(knext, kk, sn);
    float mx = -INFINITY;
#pragma unroll
    for (int v = 0; v < 16; ++v) mx = fmaxf(mx, sc[v]);
    mx = fmaxf(mx, other_half(mx)) * scale_log2;   // scale > 0
    const bool upd = mx > m_ref + 8.f;                // move the reference by > 2^8 only
    if (__ballot(upd)) {
      const float nref = upd ? mx : m_ref;
      const float alpha = upd ? __builtin_amdgcn_exp2f(m_ref - nref) : 1.f;
      l_run *= alpha;
#pragma unroll
      for (int db = 0; db < NDB; ++db)
#pragma unroll
        for (int v = 0; v < 16; ++v) o[db][v] *= alpha;
      m_ref = nref;
    }
    const float nref = m_ref == -INFINITY ? 0.f : -m_ref;
#pragma unroll
    for (int hf = 0; hf < 2; ++hf) {
      bf16x8 pg;
      float sum = 0.f;
#pragma unroll
      for (int t = 0; t < 8; ++t) {
        const float e = __builtin_amdgcn_exp2f(fmaf(sc[hf * 8 + t], scale_log2, nref));
        sum += e;
        pg[t] = (__bf16)e;
      }
      l_run += sum;
#pragma unroll
      for (int db = 0; db < NDB; ++db) {
        const unsigned char* va = vbuf + voff[db & 1] + ((16 * hf) * ROWB + 64 * (db & ~1));
        const unsigned char* vb = vbuf + voff[db & 1] + ((16 * hf + 8) * ROWB + 64 * (db & ~1));
        const bf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)va);
        const bf16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)vb);
        const bf16x8 a = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
        o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, pg, o[db], 0, 0, 0);
      }
#pragma unroll
      for (int kk = NKK / 2 + hf * (NKK / 4); kk < NKK / 2 + (hf + 1) * (NKK / 4); ++kk)
        s_mfma(knext, kk, sn);
    }
  };

  // one step for group KG: slots of stage 2t + KG (V) and 2t + 2 + KG (K look-ahead)
  f32x16 sA, sB;
  auto run = [&](auto tag) __attribute__((always_inline)) {
    constexpr int KGc = decltype(tag)::value;
    unsigned char* const ks[8] = {s_k0, s_k1, s_k2, s_k3, s_k4, s_k5, s_k6, s_k7};
    unsigned char* const vs[8] = {s_v0, s_v1, s_v2, s_v3, s_v4, s_v5, s_v6, s_v7};
    int pnext1 = 0;                   // paged: the page id of this wave's next stage
    auto step = [&](auto pt, f32x16& sc, f32x16& sn, int t) __attribute__((always_inline)) {
      constexpr int P = decltype(pt)::value;   // t % 4
      TAPS_WAIT_VMCNT(8);             // V(2t), V(2t+1), K(2t+2), K(2t+3): this wave's part
      TAPS_STAGE_BARRIER();           // ... and every other wave's part; and every wave is
                                      // done with the slots of step t - 1, refilled here
      if constexpr (PAGED) {
        const int qw = wave_u >> 1;                 // stage 2t + 6 + qw: V, V, K, K
        unsigned char* const dst = qw == 0 ? vs[(2 * P + 6) & 7] : qw == 1 ? vs[(2 * P + 7) & 7]
                                 : qw == 2 ? ks[(2 * P + 8) & 7] : ks[(2 * P + 9) & 7];
        issue4_paged(qw < 2 ? vrs : krs, dst, 2 * t + 6 + qw,
                     __builtin_amdgcn_readfirstlane(pnext1));
        pnext1 = page_of_stage(2 * t + 8 + qw);      // the next step's stage of this wave
      } else {
        issue_at(vrs, vs[(2 * P + 6) & 7], 2 * t + 6, 0);
        issue_at(vrs, vs[(2 * P + 7) & 7], 2 * t + 7, 0);
        issue_at(krs, ks[(2 * P + 8) & 7], 2 * t + 8, 0);
        issue_at(krs, ks[(2 * P + 9) & 7], 2 * t + 9, 0);
      }
      softmax_pv(sc, vs[(2 * P + KGc) & 7], ks[(2 * P + 2 + KGc) & 7], sn,
                 k_begin + (2 * t + KGc) * KT);
    };
    TAPS_WAIT_VMCNT(4);               // K(0), K(1)
    TAPS_LDS_BARRIER();               // every wave has its queries: V slots 4-7 refill below
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk) s_mfma(ks[KGc], kk, sA);
    int pg[4] = {0, 0, 0, 0};         // paged: the pages of stages 4 .. 7
    if constexpr (PAGED) {
      read_pages4(4, pg);
#pragma unroll
      for (int q = 0; q < 4; ++q) pg[q] = __builtin_amdgcn_readfirstlane(pg[q]);
      pnext1 = page_of_stage(6 + (wave_u >> 1));   // this wave's stage of the first step
    }
    issue(vrs, s_v2, 2); issue(vrs, s_v3, 3);
    issue_at(krs, s_k4, 4, pg[0]); issue_at(krs, s_k5, 5, pg[1]);
    issue_at(vrs, s_v4, 4, pg[0]); issue_at(vrs, s_v5, 5, pg[1]);
    issue_at(krs, s_k6, 6, pg[2]); issue_at(krs, s_k7, 7, pg[3]);
    for (int t = 0;;) {
      step(GroupTag<0>(), sA, sB, t);
      if (++t >= steps) break;
      step(GroupTag<1>(), sB, sA, t);
      if (++t >= steps) break;
      step(GroupTag<2>(), sA, sB, t);
      if (++t >= steps) break;
      step(GroupTag<3>(), sB, sA, t);
      if (++t >= steps) break;
    }
  };
  if (kg == 0) run(GroupTag<0>());
  else run(GroupTag<1>());
  // the look-ahead loads past the split's end read nothing from memory; let them land
  // before the slots are reused and the workgroup's LDS is released
  TAPS_WAIT_VMCNT(0);
  __syncthreads();

  const float lsum = l_run + other_half(l_run);
  // ---- merge the key groups through LDS.  Group 0 finishes head dims 0..63 and group 1
  // dims 64..127: each wave leaves the two O^T blocks the other group finishes, and its
  // (max, sum), in the K slot of its own index.
  auto xslot = [&](int w) -> float* {
    switch (w) {
      case 0: return (float*)s_k0;
      case 1: return (float*)s_k1;
      case 2: return (float*)s_k2;
      case 3: return (float*)s_k3;
      case 4: return (float*)s_k4;
      case 5: return (float*)s_k5;
      case 6: return (float*)s_k6;
      default: return (float*)s_k7;
    }
  };
  {
    // 16-byte LDS accesses: value v of block j at float4 (4 j + v / 4) of this lane
    float4* mine = (float4*)xslot(wave);
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int db = kg == 0 ? 2 + j : j;     // the blocks the other group finishes
#pragma unroll
      for (int v4 = 0; v4 < 4; ++v4)
        mine[(4 * j + v4) * 64 + lane] =
            make_float4(o[db][4 * v4], o[db][4 * v4 + 1], o[db][4 * v4 + 2], o[db][4 * v4 + 3]);
    }
    s_ml[wave * 64 + lane] = make_float2(m_ref, lsum);
  }
  __syncthreads();
  const int other = wave ^ 4;
  const float4* theirs = (const float4*)xslot(other);
  const float2 ml = s_ml[other * 64 + lane];
  const float M = fmaxf(m_ref, ml.x);
  const float a0 = m_ref == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m_ref - M);
  const float a1 = ml.x == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(ml.x - M);
  const float Ls = lsum * a0 + ml.y * a1;
  const float inv = Ls > 0.f ? 1.f / Ls : 0.f;

  // ---- write this split's partial: O / sum in bf16 for this group's 64 head dims of the
  // wave's 32 rows, max and sum.  The tile goes through LDS (this wave's V slot, free
  // now) so that each store instruction writes whole 128-byte row segments.  The stores
  // are non-temporal: only the combine, a later launch, reads the partials, and streaming
  // them out of the L2 leaves less to write back when the kernel ends (measured: the
  // kernel took 0.5 us less at the Qwen3-8B shape).
  constexpr int TROW = 144;            // bytes per staged row (128 + 16: fewer bank conflicts)
  unsigned char* stage;
  switch (wave) {
    case 0: stage = s_v0; break;
    case 1: stage = s_v1; break;
    case 2: stage = s_v2; break;
    case 3: stage = s_v3; break;
    case 4: stage = s_v4; break;
    case 5: stage = s_v5; break;
    case 6: stage = s_v6; break;
    default: stage = s_v7; break;
  }
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int db = kg == 0 ? j : 2 + j;       // the blocks this group finishes
#pragma unroll
    for (int r4 = 0; r4 < 4; ++r4) {
      const float4 th = theirs[(4 * j + r4) * 64 + lane];
      const float tv[4] = {th.x, th.y, th.z, th.w};
      float x[4];
#pragma unroll
      for (int t = 0; t < 4; ++t) x[t] = (o[db][4 * r4 + t] * a0 + tv[t] * a1) * inv;
      *(uint2*)(stage + l32 * TROW + 2 * (j * 32 + 8 * r4 + 4 * hl)) = pack_bf16x4(x[0], x[1], x[2], x[3]);
    }
  }
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  const size_t obase = (size_t)pair * mrows_pad;
  const int qbase = row0 + rg * 32;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int r = 8 * i + (lane >> 3), c = (lane & 7) * 16;   // row in the tile, byte in the half
    const i32x4 v = *(const i32x4*)(stage + r * TROW + c);
    __builtin_nontemporal_store(v, (i32x4*)((unsigned char*)(wsO + (obase + qbase + r) * HD) + kg * 128 + c));
  }
  const int qr = qbase + l32;
  if (kg == 0 && hl == 0) {
    f32x2 ml2;
    ml2.x = M;
    ml2.y = Ls;
    __builtin_nontemporal_store(ml2, (f32x2*)(wsML + obase + qr));
  }
}
#endif

// Contiguous cache: the kernel keeps exactly the arguments it had before the paged mode
// existed (a longer argument block measured 0.3 us slower per launch, same code).
__global__ __launch_bounds__(512) void attn_bf16_kernel(
    const uint16_t* __restrict__ Q, const uint16_t* __restrict__ Kc,
    const uint16_t* __restrict__ Vc, const int64_t* __restrict__ offp,
    const int32_t* __restrict__ ctxp, const int32_t* __restrict__ parentp,
    const int32_t* __restrict__ nnp, int N, int Hq, int Hkv, int max_ctx, float scale_log2,
    int split_len, int splits, int mtiles, int pairs, int mrows_pad, uint16_t* __restrict__ wsO,
    float2* __restrict__ wsML, DivMagic dm, int batch, int target_pairs, int lcap,
    int2* __restrict__ tab) {
#if defined(__HIP_DEVICE_COMPILE__)
  attn_bf16_body<false>(Q, Kc, Vc, offp, ctxp, parentp, nnp, N, Hq, Hkv, max_ctx, scale_log2, split_len,
                       splits, mtiles, pairs, mrows_pad, wsO, wsML, dm, batch, target_pairs, lcap,
                       tab, PagedKV{nullptr, 0, 1, 5});
#endif
}

// Paged cache (C20 of the readings: tree_verify_attn_paged)
__global__ __launch_bounds__(512) void attn_bf16_paged_kernel(
    const uint16_t* __restrict__ Q, const uint16_t* __restrict__ Kc,
    const uint16_t* __restrict__ Vc, const int64_t* __restrict__ offp,
    const int32_t* __restrict__ ctxp, const int32_t* __restrict__ parentp,
    const int32_t* __restrict__ nnp, int N, int Hq, int Hkv, int max_ctx, float scale_log2,
    int split_len, int splits, int mtiles, int pairs, int mrows_pad, uint16_t* __restrict__ wsO,
    float2* __restrict__ wsML, DivMagic dm, int batch, int target_pairs, int lcap,
    int2* __restrict__ tab, PagedKV pk) {
#if defined(__HIP_DEVICE_COMPILE__)
  attn_bf16_body<true>(Q, Kc, Vc, offp, ctxp, parentp, nnp, N, Hq, Hkv, max_ctx, scale_log2, split_len,
                       splits, mtiles, pairs, mrows_pad, wsO, wsML, dm, batch, target_pairs, lcap,
                       tab, pk);
#endif
}

// Split combine: grid (row blocks, batch); one thread per 8 head dims of one output row
// (16-byte loads and stores).  CH = splits merged per group: the plan's split count for one
// request (up to 16), 4 for the ragged list, whose requests mostly hold a few splits each.
// Workgroups of 128 threads (8 rows of head_dim 128): the Qwen3-8B round's 2048 rows then
// spread over 256 workgroups, one per CU, and each CU pulls half as many partials (the
// combine took 4.7 us against 5.0 us with 256 threads).
constexpr int kCombineThreads = 128;
template <int HD, int CH>
__global__ __launch_bounds__(kCombineThreads) void attn_combine_kernel(
    const uint16_t* __restrict__ wsO, const float2* __restrict__ wsML,
    const int32_t* __restrict__ ctxp, const int32_t* __restrict__ nnp, int N, int Hq, int Hkv,
    int max_ctx, int split_len, int splits, int mrows_pad, DivMagic dm,
    uint16_t* __restrict__ O, const int2* __restrict__ tab, int batch) {
  constexpr int TPR = HD / 8;  // threads per output row, 8 values each
  constexpr int RPB = kCombineThreads / TPR;
  asm volatile("" ::"s"(wsO), "s"(wsML), "s"(ctxp), "s"(nnp), "s"(N), "s"(Hq), "s"(Hkv),
               "s"(max_ctx), "s"(split_len), "s"(splits), "s"(mrows_pad), "s"(dm.hk),
               "s"(dm.g), "s"(O), "s"(tab), "s"(batch));
  const int b = blockIdx.y;
  const int rr = blockIdx.x * RPB + threadIdx.x / TPR;   // (node, query head) of request b
  const int d = (threadIdx.x % TPR) * 8;
  if (rr >= N * Hq) return;
  const int i = dm.div(rr, Hq, dm.hk), hq = rr - i * Hq;   // dm.hk holds the Hq multiplier
  const int G = Hq / Hkv, g = dm.div(hq, G, dm.g);
  const int qr = i * G + (hq - g * G);
  // the request's splits of KV head g: slots base .. base + cap - 1 (the ragged list's
  // table, written by the attention kernel, or the host's fixed split count)
  size_t base;
  int cap;
  if (tab != nullptr) {
    const int2 t = tab[b];
    base = (size_t)t.x + (size_t)g * t.y;
    cap = t.y;
    split_len = tab[batch].x;
  } else {
    base = (size_t)(b * Hkv + g) * splits;
    cap = splits;
  }
  // each split holds O_s / l_s (bf16) and (m_s, l_s) with m_s in base 2:
  // O = sum_s 2^(m_s - M) l_s (O_s / l_s) / sum_s 2^(m_s - M) l_s.  The loads of the first
  // CH splits go out before the request's sizes are known (their addresses do not depend on
  // them; splits past the request's keys are masked once the sizes have arrived), then
  // groups of up to CH splits are merged with a running maximum.
  float2 ml[CH];
  uint4 ov[CH];
  auto load_group = [&](int s0) __attribute__((always_inline)) {
#pragma unroll
    for (int t = 0; t < CH; ++t) {
      const size_t r = (base + min(s0 + t, cap - 1)) * mrows_pad + qr;
      ml[t] = wsML[r];
      ov[t] = *(const uint4*)(wsO + r * HD + d);
    }
  };
  if (cap > 0) load_group(0);
  int ctx_raw, n_raw;
  load_two_scalars(ctxp + b, nnp + b, ctx_raw, n_raw);
  const int n = min(max(n_raw, 0), N);
  if (i >= n) return;
  const int ctx = min(max(ctx_raw, 0), max_ctx);
  const int R = ctx + n;
  const int nspl = min((R + split_len - 1) / split_len, cap);
  float M = -INFINITY, L = 0.f;
  float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  for (int s0 = 0; s0 < nspl; s0 += CH) {
    if (s0 > 0) load_group(s0);
    // splits past the request's keys were not written by this call: their slots hold
    // whatever the workspace held before (possibly NaN bits), so values and weights are
    // both replaced, not multiplied by a zero weight
#pragma unroll
    for (int t = 0; t < CH; ++t)
      if (s0 + t >= nspl) {
        ml[t] = make_float2(-INFINITY, 0.f);
        ov[t] = make_uint4(0u, 0u, 0u, 0u);
      }
    float Mc = M;
#pragma unroll
    for (int t = 0; t < CH; ++t) Mc = fmaxf(Mc, ml[t].x);
    if (Mc == -INFINITY) continue;
    const float a = M == -INFINITY ? 0.f : exp2f(M - Mc);
    L *= a;
#pragma unroll
    for (int k = 0; k < 8; ++k) acc[k] *= a;
#pragma unroll
    for (int t = 0; t < CH; ++t) {
      const float w = ml[t].x == -INFINITY ? 0.f : exp2f(ml[t].x - Mc) * ml[t].y;
      L += w;
      const uint32_t wd[4] = {ov[t].x, ov[t].y, ov[t].z, ov[t].w};
#pragma unroll
      for (int k = 0; k < 4; ++k) {
        acc[2 * k] += w * __uint_as_float(wd[k] << 16);
        acc[2 * k + 1] += w * __uint_as_float(wd[k] & 0xFFFF0000u);
      }
    }
    M = Mc;
  }
  const float inv = 1.f / L;
  const uint2 lo = pack_bf16x4(acc[0] * inv, acc[1] * inv, acc[2] * inv, acc[3] * inv);
  const uint2 hi = pack_bf16x4(acc[4] * inv, acc[5] * inv, acc[6] * inv, acc[7] * inv);
  *(uint4*)(O + (((size_t)b * N + i) * Hq + hq) * HD + d) = make_uint4(lo.x, lo.y, hi.x, hi.y);
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
  __shared__ uint64_t s_anc[kAncWords];
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
    uint64_t a[kAncWords];
    const int32_t* pp = parentp + (size_t)b * N;
    ancestor_mask(i, [&](int j) { return pp[j]; }, a);
    for (int w = 0; w < kAncWords; ++w) s_anc[w] = a[w];
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
      ok = (s_anc[t >> 6] >> (t & 63)) & 1ull;
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

AttnPlan plan_attn(int batch, int budget, int Hq, int Hkv, int head_dim, int max_ctx,
                   int max_len) {
  AttnPlan p;
  const int G = Hq / Hkv;
  const int mrows = budget * G;
  p.qb = 1;
  p.wk = 1;
  p.mtile = 4 * 32;
  p.mtiles = (mrows + p.mtile - 1) / p.mtile;
  p.ragged = 0;
  p.target_pairs = p.pairs_max = 0;
  // the buffer ranges of a split, look-ahead included, stay below 2^31 bytes
  const long long rsb0 = (long long)Hkv * head_dim * 2;
  p.lcap = (int)((((1ll << 31) - 1) / rsb0 - 5 * kKT) / kKT * kKT);
  if (max_len > 0 && max_len < p.lcap) p.lcap = max_len / kKT * kKT;

  // Split the keys so that the workgroups (one per CU: the K/V rings fill its LDS) finish
  // soonest: estimated time = rounds of 256 workgroups x (32-key stages per split + ~8
  // stages' worth of prologue and partial writes).  Rounding the split count up to fill
  // the chip can leave a second round of a few workgroups that doubles the time.
  const int keys = max_ctx + budget;
  const int step = kKT;
  const long long base = (long long)batch * Hkv * p.mtiles;
  int splits = 1;
  long long best = -1;
  for (int s = 1; s <= 64; ++s) {
    int l = (keys + s - 1) / s;
    l = ((l + step - 1) / step) * step;
    if (l < 2 * step) l = 2 * step;
    const long long rounds = (base * s + 255) / 256;
    const long long cost = rounds * (l / step + 8);
    if (best < 0 || cost < best) {
      best = cost;
      splits = s;
    }
  }
  int len = (keys + splits - 1) / splits;
  len = ((len + step - 1) / step) * step;
  if (len < 2 * step) len = 2 * step;
  if (len > p.lcap) len = p.lcap;
  p.split_len = len;
  p.splits = (keys + len - 1) / len;
  if (batch > 1 && head_dim == 128) {
    // Several requests: their lengths are known only on the device, where the kernel picks
    // the split length (ragged_pick): this plan's for lengths close to each other, else one
    // sized for about three workgroups per CU over the batch's actual keys (measured: a
    // 16-request batch with lengths from 512 to 16K keys takes 12 % less time than with
    // every request split for max_ctx, a 4 x 32K batch the same).
    const int target = (3 * 256 + p.mtiles - 1) / p.mtiles;
    const long long worst = ((long long)batch * (max_ctx + budget) * Hkv + target - 1) / target;
    const long long pm = std::max((long long)target + (long long)batch * Hkv,
                                  (long long)batch * Hkv * p.splits);
    if (worst <= p.lcap && pm < (1ll << 24)) {
      p.ragged = 1;
      p.target_pairs = target;
      p.pairs_max = (int)pm;
    }
  }
  return p;
}

// split partials [slot][mtiles * mtile][head_dim] bf16, then their (max, sum) pairs, then
// (ragged list) the per-request table of the combine
static size_t attn_rows(const AttnPlan& pl, int batch, int Hkv) {
  const size_t slots = pl.ragged ? (size_t)pl.pairs_max : (size_t)batch * Hkv * pl.splits;
  return slots * (size_t)pl.mtiles * pl.mtile;
}
static size_t attn_tab_offset(const AttnPlan& pl, int batch, int Hkv, int head_dim) {
  const size_t rows = attn_rows(pl, batch, Hkv);
  return (rows * head_dim * sizeof(uint16_t) + rows * sizeof(float2) + 15) & ~(size_t)15;
}

size_t attn_ws_bytes(const AttnPlan& pl, int batch, int /*budget*/, int /*Hq*/, int Hkv,
                     int head_dim) {
  return attn_tab_offset(pl, batch, Hkv, head_dim) +
         (pl.ragged ? (size_t)(batch + 1) * sizeof(int2) : 0) + 256;
}

// The bf16 attention and its split combine; PAGED takes K and V from page pools through
// the block table of pk (head_dim 128 only), else from the contiguous cache at off[b]
template <bool PAGED>
static hipError_t launch_attn_bf16_impl(const void* Q, const void* K, const void* V,
                                        const int64_t* off, const PagedKV& pk,
                                        const int32_t* ctx, const int32_t* parent,
                                        const int32_t* n, int batch, int budget, int Hq, int Hkv,
                                        int head_dim, int max_ctx, float scale,
                                        const AttnPlan& pl, void* O, void* ws, hipStream_t s,
                                        hipEvent_t ev_begin, hipEvent_t ev_end) {
  if (batch <= 0) return hipSuccess;
  const int mrows_pad = pl.mtiles * pl.mtile;
  const size_t rows = attn_rows(pl, batch, Hkv);
  uint16_t* wsO = (uint16_t*)ws;
  float2* wsML = (float2*)((char*)ws + rows * head_dim * sizeof(uint16_t));
  int2* tab = pl.ragged ? (int2*)((char*)ws + attn_tab_offset(pl, batch, Hkv, head_dim)) : nullptr;
  const int pairs = pl.ragged ? pl.pairs_max : pl.splits * batch * Hkv;
  dim3 grid((unsigned)(8 * pl.mtiles * ((pairs + 7) / 8)));
  dim3 block(256u);
  const float sl2 = scale * kLog2e;
  const uint16_t *q = (const uint16_t*)Q, *k = (const uint16_t*)K, *v = (const uint16_t*)V;
  // with events, the launch records the kernel's own start and end (hipExtLaunchKernel)
  if (head_dim == 128) {
    const dim3 block8(512u);
    const DivMagic dm{DivMagic::make(pl.mtiles), DivMagic::make(pl.splits), DivMagic::make(Hkv),
                      DivMagic::make(Hq / Hkv)};
    if constexpr (PAGED) {
      if (ev_begin || ev_end)
        hipExtLaunchKernelGGL(attn_bf16_paged_kernel, grid, block8, 0, s, ev_begin, ev_end, 0,
                              q, k, v, off, ctx, parent, n, budget, Hq, Hkv, max_ctx, sl2,
                              pl.split_len, pl.splits, pl.mtiles, pairs, mrows_pad, wsO, wsML,
                              dm, batch, pl.target_pairs, pl.lcap, tab, pk);
      else
        attn_bf16_paged_kernel<<<grid, block8, 0, s>>>(
            q, k, v, off, ctx, parent, n, budget, Hq, Hkv, max_ctx, sl2, pl.split_len, pl.splits,
            pl.mtiles, pairs, mrows_pad, wsO, wsML, dm, batch, pl.target_pairs, pl.lcap, tab, pk);
    } else {
      if (ev_begin || ev_end)
        hipExtLaunchKernelGGL(attn_bf16_kernel, grid, block8, 0, s, ev_begin, ev_end, 0, q, k,
                              v, off, ctx, parent, n, budget, Hq, Hkv, max_ctx, sl2,
                              pl.split_len, pl.splits, pl.mtiles, pairs, mrows_pad, wsO, wsML,
                              dm, batch, pl.target_pairs, pl.lcap, tab);
      else
        attn_bf16_kernel<<<grid, block8, 0, s>>>(q, k, v, off, ctx, parent, n, budget, Hq, Hkv,
                                                 max_ctx, sl2, pl.split_len, pl.splits,
                                                 pl.mtiles, pairs, mrows_pad, wsO, wsML, dm,
                                                 batch, pl.target_pairs, pl.lcap, tab);
    }
  } else if constexpr (!PAGED) {
    if (ev_begin || ev_end)
      hipExtLaunchKernelGGL(attn_bf16_w4_kernel<64>, grid, block, 0, s, ev_begin, ev_end, 0, q,
                            k, v, off, ctx, parent, n, budget, Hq, Hkv, max_ctx, sl2,
                            pl.split_len, pl.splits, pl.mtiles, pairs, mrows_pad, wsO, wsML);
    else
      attn_bf16_w4_kernel<64><<<grid, block, 0, s>>>(q, k, v, off, ctx, parent, n, budget, Hq,
                                                     Hkv, max_ctx, sl2, pl.split_len,
                                                     pl.splits, pl.mtiles, pairs, mrows_pad,
                                                     wsO, wsML);
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int rows_req = budget * Hq;   // output rows of one request
  const DivMagic cm{0u, 0u, DivMagic::make(Hq), DivMagic::make(Hq / Hkv)};
  // splits per group: the one-request plan's split count (rounded up to 4, 8 or 16), 4
  // for the ragged list
  const int ch = tab != nullptr || pl.splits <= 4 ? 4 : pl.splits <= 8 ? 8 : 16;
  const int2* tb = head_dim == 128 ? tab : nullptr;
#define TAPS_COMBINE(HDC, CHC)                                                               \
  attn_combine_kernel<HDC, CHC>                                                              \
      <<<dim3((unsigned)((rows_req + kCombineThreads / (HDC / 8) - 1) /                      \
                         (kCombineThreads / (HDC / 8))),                                      \
              (unsigned)batch),                                                              \
         dim3(kCombineThreads), 0, s>>>(wsO, wsML, ctx, n, budget, Hq, Hkv, max_ctx,          \
                                        pl.split_len, pl.splits, mrows_pad, cm, (uint16_t*)O, \
                                        tb, batch)
  if (head_dim == 128) {
    if (ch == 4) TAPS_COMBINE(128, 4);
    else if (ch == 8) TAPS_COMBINE(128, 8);
    else TAPS_COMBINE(128, 16);
  } else {
    if (ch == 4) TAPS_COMBINE(64, 4);
    else if (ch == 8) TAPS_COMBINE(64, 8);
    else TAPS_COMBINE(64, 16);
  }
#undef TAPS_COMBINE
  return hipGetLastError();
}

hipError_t launch_attn_bf16(const void* Q, const void* K, const void* V, const int64_t* off,
                            const int32_t* ctx, const int32_t* parent, const int32_t* n,
                            int batch, int budget, int Hq, int Hkv, int head_dim, int max_ctx,
                            float scale, const AttnPlan& pl, void* O, void* ws, hipStream_t s,
                            hipEvent_t ev_begin, hipEvent_t ev_end) {
  return launch_attn_bf16_impl<false>(Q, K, V, off, PagedKV{nullptr, 0, 1, 5}, ctx, parent, n,
                                      batch, budget, Hq, Hkv, head_dim, max_ctx, scale, pl, O,
                                      ws, s, ev_begin, ev_end);
}

hipError_t launch_attn_bf16_paged(const void* Q, const void* K_pages, const void* V_pages,
                                  const int32_t* block_table, int max_pages, int num_pages,
                                  int page_shift, const int32_t* ctx, const int32_t* parent,
                                  const int32_t* n, int batch, int budget, int Hq, int Hkv,
                                  int max_ctx, float scale, const AttnPlan& pl, void* O,
                                  void* ws, hipStream_t s, hipEvent_t ev_begin,
                                  hipEvent_t ev_end) {
  return launch_attn_bf16_impl<true>(Q, K_pages, V_pages, nullptr,
                                     PagedKV{block_table, max_pages, num_pages, page_shift}, ctx,
                                     parent, n, batch, budget, Hq, Hkv, 128, max_ctx, scale, pl,
                                     O, ws, s, ev_begin, ev_end);
}

int paged_max_split(int page_shift) { return (kPageSlots - 1) << page_shift; }

hipError_t launch_attn_f32(const float* Q, const float* K, const float* V, const int64_t* off,
                           const int32_t* ctx, const int32_t* parent, const int32_t* n,
                           int batch, int budget, int Hq, int Hkv, int head_dim, int max_ctx,
                           float scale, float* O, hipStream_t s, hipEvent_t ev_begin,
                           hipEvent_t ev_end) {
  if (batch <= 0) return hipSuccess;
  dim3 grid((unsigned)budget, (unsigned)Hq, (unsigned)batch), block(kThreads);
  if (head_dim == 128)
    hipExtLaunchKernelGGL(attn_f32_kernel<128>, grid, block, 0, s, ev_begin, ev_end, 0, Q, K, V,
                          off, ctx, parent, n, budget, Hq, Hkv, max_ctx, scale, O);
  else
    hipExtLaunchKernelGGL(attn_f32_kernel<64>, grid, block, 0, s, ev_begin, ev_end, 0, Q, K, V,
                          off, ctx, parent, n, budget, Hq, Hkv, max_ctx, scale, O);
  return hipGetLastError();
}

}  // namespace taps
