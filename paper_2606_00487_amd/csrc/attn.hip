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
#include "common.h"

namespace taps {

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int kThreads = 256;
constexpr int kWavesA = 4;
constexpr int kKT = 64;  // keys per tile
constexpr float kLog2e = 1.4426950408889634f;

__device__ inline int swz_v(int d) { return (d ^ (d >> 3)) & 7; }

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

template <int QB, int HD>
__global__ __launch_bounds__(kThreads) void attn_bf16_kernel(
    const uint16_t* __restrict__ Q, const uint16_t* __restrict__ Kc,
    const uint16_t* __restrict__ Vc, const int64_t* __restrict__ offp,
    const int32_t* __restrict__ ctxp, const int32_t* __restrict__ parentp,
    const int32_t* __restrict__ nnp, int N, int Hq, int Hkv, int max_ctx, float scale_log2,
    int split_len, int splits, int mrows_pad, float* __restrict__ wsO,
    float2* __restrict__ wsML) {
  constexpr int DC = HD / 8;          // 16-byte chunks per K/V row
  constexpr int MT = kWavesA * 32 * QB;
  constexpr int NDB = HD / 32;        // 32-row blocks of O^T
  constexpr int NKK = HD / 16;        // MFMA k-steps over head_dim
  __shared__ __attribute__((aligned(16))) uint16_t s_k[kKT * HD];
  __shared__ __attribute__((aligned(16))) uint16_t s_vt[HD * kKT];
  __shared__ uint64_t s_anc[TAPS_MAX_BUDGET][4];
  __shared__ int s_par[TAPS_MAX_BUDGET];

  const int split = blockIdx.x, mt = blockIdx.y, bg = blockIdx.z;
  const int b = bg / Hkv, g = bg - (bg / Hkv) * Hkv;
  const int G = Hq / Hkv;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int l32 = lane & 31, hl = lane >> 5;

  const int ctx = min(max(ctxp[b], 0), max_ctx);
  const int n = min(max(nnp[b], 0), N);
  const int R = ctx + n;
  const int k_begin = split * split_len;
  const int k_end = min(R, k_begin + split_len);
  const int row0 = mt * MT;
  if (k_begin >= k_end || row0 >= n * G) return;
  const int64_t kv0 = offp[b];

  // ---- queries of this lane (B operand of S^T = K Q^T)
  bf16x8 q[QB][NKK];
  int qnode[QB];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    int qr = row0 + wave * 32 * QB + qb * 32 + l32;
    qr = min(qr, N * G - 1);
    const int node = qr / G, hq = g * G + (qr - node * G);
    qnode[qb] = node;
    const uint16_t* qp = Q + (((size_t)b * N + node) * Hq + hq) * HD;
#pragma unroll
    for (int kk = 0; kk < NKK; ++kk) q[qb][kk] = *(const bf16x8*)(qp + kk * 16 + hl * 8);
  }

  // ---- ancestor masks, only when this split reaches the tree rows
  const bool tree_part = k_end > ctx;
  uint64_t anc[QB][4];
  if (tree_part) {
    for (int i = tid; i < n; i += kThreads) s_par[i] = parentp[(size_t)b * N + i];
    __syncthreads();
    for (int i = tid; i < n; i += kThreads) {
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

  f32x16 o[NDB][QB];
#pragma unroll
  for (int db = 0; db < NDB; ++db)
#pragma unroll
    for (int qb = 0; qb < QB; ++qb)
#pragma unroll
      for (int v = 0; v < 16; ++v) o[db][qb][v] = 0.f;
  float m_run[QB], l_run[QB];
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) { m_run[qb] = -INFINITY; l_run[qb] = 0.f; }

  const size_t row_stride = (size_t)Hkv * HD;  // elements between consecutive cache rows
  const uint16_t* kbase = Kc + (size_t)kv0 * row_stride + (size_t)g * HD;
  const uint16_t* vbase = Vc + (size_t)kv0 * row_stride + (size_t)g * HD;

  for (int k0 = k_begin; k0 < k_end; k0 += kKT) {
    // ---- stage K (row-major, chunk-swizzled) and V^T (transposed, permuted keys)
#pragma unroll
    for (int c = 0; c < kKT * DC / kThreads; ++c) {
      const int id = tid + kThreads * c;
      const int kr = id / DC, dc = id - (id / DC) * DC;
      uint4 w = {0u, 0u, 0u, 0u};
      if (k0 + kr < k_end) w = *(const uint4*)(kbase + (size_t)(k0 + kr) * row_stride + dc * 8);
      *(uint4*)(s_k + kr * HD + ((dc ^ (kr & 7)) * 8)) = w;
    }
    if (tid < 16 * DC) {
      const int a = tid / DC, dc = tid - (tid / DC) * DC;
      uint4 w[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int kr = 4 * a + j;
        w[j] = make_uint4(0u, 0u, 0u, 0u);
        if (k0 + kr < k_end) w[j] = *(const uint4*)(vbase + (size_t)(k0 + kr) * row_stride + dc * 8);
      }
      const int as = a & 7;
      const int pos = 32 * (a >> 3) + ((as & 1) << 4) + ((as >> 1) << 2);
      const int chunk = pos >> 3, half = (pos >> 2) & 1;
#pragma unroll
      for (int dd = 0; dd < 8; ++dd) {
        const int d = dc * 8 + dd;
        const int sh = (dd & 1) * 16;
        uint32_t e[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const uint32_t ww = dd < 2 ? w[j].x : dd < 4 ? w[j].y : dd < 6 ? w[j].z : w[j].w;
          e[j] = (ww >> sh) & 0xFFFFu;
        }
        uint2 pk;
        pk.x = e[0] | (e[1] << 16);
        pk.y = e[2] | (e[3] << 16);
        *(uint2*)(s_vt + d * kKT + ((chunk ^ swz_v(d)) * 8) + half * 4) = pk;
      }
    }
    __syncthreads();

    // ---- S^T = K Q^T for the two 32-key blocks
    f32x16 s[2][QB];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
#pragma unroll
      for (int qb = 0; qb < QB; ++qb)
#pragma unroll
        for (int v = 0; v < 16; ++v) s[kb][qb][v] = 0.f;
      const int kr = kb * 32 + l32;
#pragma unroll
      for (int kk = 0; kk < NKK; ++kk) {
        const bf16x8 a = *(const bf16x8*)(s_k + kr * HD + (((2 * kk + hl) ^ (kr & 7)) * 8));
#pragma unroll
        for (int qb = 0; qb < QB; ++qb)
          s[kb][qb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, q[qb][kk], s[kb][qb], 0, 0, 0);
      }
    }

    // ---- mask, online softmax (base 2), P^T in bf16
    bf16x8 p[2][QB][2];
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      float mx = -INFINITY;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int key = k0 + kb * 32 + 8 * (v >> 2) + 4 * hl + (v & 3);
          bool ok = key < k_end;
          if (key >= ctx) {
            const int t = key - ctx;
            ok = ok && ((mask_word(anc[qb], (t >> 6) & 3) >> (t & 63)) & 1ull);
          }
          const float x = ok ? s[kb][qb][v] * scale_log2 : -INFINITY;
          s[kb][qb][v] = x;
          mx = fmaxf(mx, x);
        }
      mx = fmaxf(mx, __shfl_xor(mx, 32));
      const float m_new = fmaxf(m_run[qb], mx);
      const float ref = m_new == -INFINITY ? 0.f : m_new;
      const float alpha = exp2f(m_run[qb] - ref);
      float sum = 0.f;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int hf = 0; hf < 2; ++hf) {
          bf16x8 pk;
#pragma unroll
          for (int t = 0; t < 8; ++t) {
            const float e = exp2f(s[kb][qb][hf * 8 + t] - ref);
            sum += e;
            pk[t] = (__bf16)e;
          }
          p[kb][qb][hf] = pk;
        }
      l_run[qb] = l_run[qb] * alpha + sum;
      m_run[qb] = m_new;
#pragma unroll
      for (int db = 0; db < NDB; ++db)
#pragma unroll
        for (int v = 0; v < 16; ++v) o[db][qb][v] *= alpha;
    }

    // ---- O^T += V^T P^T
#pragma unroll
    for (int db = 0; db < NDB; ++db) {
      const int d = db * 32 + l32;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int hf = 0; hf < 2; ++hf) {
          const int chunk = 4 * kb + 2 * hl + hf;
          const bf16x8 a = *(const bf16x8*)(s_vt + d * kKT + ((chunk ^ swz_v(d)) * 8));
#pragma unroll
          for (int qb = 0; qb < QB; ++qb)
            o[db][qb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, p[kb][qb][hf], o[db][qb], 0, 0, 0);
        }
    }
    __syncthreads();
  }

  // ---- write this split's unnormalised partial output, max and sum
  const size_t base = ((size_t)bg * splits + split) * mrows_pad;
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    const int qr = row0 + wave * 32 * QB + qb * 32 + l32;
    const float lsum = l_run[qb] + __shfl_xor(l_run[qb], 32);
    float* op = wsO + (base + qr) * HD;
#pragma unroll
    for (int db = 0; db < NDB; ++db)
#pragma unroll
      for (int r4 = 0; r4 < 4; ++r4) {
        const int d = db * 32 + 8 * r4 + 4 * hl;
        *(float4*)(op + d) = make_float4(o[db][qb][4 * r4], o[db][qb][4 * r4 + 1],
                                         o[db][qb][4 * r4 + 2], o[db][qb][4 * r4 + 3]);
      }
    if (hl == 0) wsML[base + qr] = make_float2(m_run[qb], lsum);
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
  float M = -INFINITY;
  for (int s = 0; s < nspl; ++s) M = fmaxf(M, wsML[(base + s) * mrows_pad + qr].x);
  float L = 0.f;
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int s = 0; s < nspl; ++s) {
    const float2 ml = wsML[(base + s) * mrows_pad + qr];
    const float w = exp2f(ml.x - M);
    L += w * ml.y;
    const float4 v = *(const float4*)(wsO + ((base + s) * mrows_pad + qr) * HD + d);
    acc.x += w * v.x; acc.y += w * v.y; acc.z += w * v.z; acc.w += w * v.w;
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
  p.qb = mrows > 128 ? 2 : 1;
  p.mtile = kWavesA * 32 * p.qb;
  p.mtiles = (mrows + p.mtile - 1) / p.mtile;
  // split the keys so that roughly 256-512 workgroups run, with at least 4 tiles each
  const int keys = max_ctx + budget;
  const long long base = (long long)batch * Hkv * p.mtiles;
  int splits = (int)((512 + base - 1) / base);
  int len = (keys + splits - 1) / splits;
  len = ((len + kKT - 1) / kKT) * kKT;
  if (len < 4 * kKT) len = 4 * kKT;
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
  dim3 grid((unsigned)pl.splits, (unsigned)pl.mtiles, (unsigned)(batch * Hkv)), block(kThreads);
  const float sl2 = scale * kLog2e;
  const uint16_t *q = (const uint16_t*)Q, *k = (const uint16_t*)K, *v = (const uint16_t*)V;
  if (ev_begin && hipEventRecord(ev_begin, s) != hipSuccess) return hipErrorInvalidValue;
#define TAPS_ATT(QB, HD)                                                                       \
  attn_bf16_kernel<QB, HD><<<grid, block, 0, s>>>(q, k, v, off, ctx, parent, n, budget, Hq, Hkv, \
                                                  max_ctx, sl2, pl.split_len, pl.splits,       \
                                                  mrows_pad, wsO, wsML)
  if (head_dim == 128) {
    if (pl.qb == 2) TAPS_ATT(2, 128); else TAPS_ATT(1, 128);
  } else {
    if (pl.qb == 2) TAPS_ATT(2, 64); else TAPS_ATT(1, 64);
  }
#undef TAPS_ATT
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (ev_end && hipEventRecord(ev_end, s) != hipSuccess) return hipErrorInvalidValue;
  const int rows_out = batch * budget * Hq;
  if (head_dim == 128) {
    const int rpb = kThreads / 32;
    attn_combine_kernel<128><<<dim3((unsigned)((rows_out + rpb - 1) / rpb)), block, 0, s>>>(
        wsO, wsML, ctx, n, batch, budget, Hq, Hkv, max_ctx, pl.split_len, pl.splits, mrows_pad,
        (uint16_t*)O);
  } else {
    const int rpb = kThreads / 16;
    attn_combine_kernel<64><<<dim3((unsigned)((rows_out + rpb - 1) / rpb)), block, 0, s>>>(
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
