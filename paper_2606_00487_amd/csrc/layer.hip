// One attention layer of the target over the draft tree (the layer slice of the
// verification forward; Sec. 4.1 stage 3 and Sec. 4.3 run the target over the selected
// tree with tree attention), bf16 storage with fp32 accumulation.  Three kernels besides
// the tree attention of attn.hip:
//
//   gemm_kernel       Y_part = X W^T for a skinny X (the budget's nodes) and a large
//                     row-major weight [N][K]: HBM-bound on the weight, which is read once.
//                     A workgroup owns 32 output columns, 64 rows and one split of K; each
//                     of its four waves takes a quarter of that split on
//                     v_mfma_f32_32x32x16_bf16, and the waves' partials are added in LDS
//                     in a fixed order.  Split partials (fp32) are added by the consumer.
//   qkv_rope_kernel   adds the projection's split partials, applies the per-head RMSNorm
//                     and the rotary embedding at position ctx + depth, and stores Q and the
//                     cache rows ctx + i of K and V in bf16.
//   reduce_kernel     adds the output projection's split partials and rounds to bf16.
#include "common.h"

namespace taps {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

__device__ inline uint16_t f32_to_bf16(float f) {   // round to nearest even
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7FFFFFFFu) > 0x7F800000u) return 0x7FC0;
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}
__device__ inline float bf16_to_f32(uint16_t h) { return __uint_as_float((uint32_t)h << 16); }

// Column segments of the weight: columns [0, end0) come from w0, [end0, end1) from w1 and
// [end1, N) from w2 (each a row-major [columns][K] array).
struct WSeg {
  const uint16_t* w0;
  const uint16_t* w1;
  const uint16_t* w2;
  int end0, end1;
};

template <int U, int NB>
__global__ __launch_bounds__(256) void gemm_kernel(const uint16_t* __restrict__ X, int M, int K,
                                                   WSeg ws, int N, int splits,
                                                   float* __restrict__ part) {
  __shared__ float red[4][2][16][kWave];
  const int c0 = blockIdx.x * 32 * NB, split = blockIdx.y, m0 = blockIdx.z * 64;
  const uint16_t* W = c0 < ws.end0 ? ws.w0 + (size_t)c0 * K
                      : c0 < ws.end1 ? ws.w1 + (size_t)(c0 - ws.end0) * K
                                     : ws.w2 + (size_t)(c0 - ws.end1) * K;
  const int tid = threadIdx.x, lane = tid & (kWave - 1), wave = tid / kWave;
  const int l32 = lane & 31, hl = lane >> 5;
  const int kper = K / (splits * 4);                 // K values per wave, a multiple of 32 U
  const int kb = split * (K / splits) + wave * kper + 8 * hl;
  // MFMA operands: lane (l32, hl) holds 8 consecutive K values at 8 hl of each 16-value
  // step, of output row l32 (X) and of output column l32 of each 32-column block (W);
  // rows past M repeat row M-1
  const uint16_t* wp = W + (size_t)l32 * K + kb;
  const size_t wnb = (size_t)32 * K;                 // next 32-column block
  const uint16_t* x0 = X + (size_t)min(m0 + l32, M - 1) * K + kb;
  const uint16_t* x1 = X + (size_t)min(m0 + 32 + l32, M - 1) * K + kb;
  f32x16 acc[2][NB];
#pragma unroll
  for (int r = 0; r < 2; ++r)
#pragma unroll
    for (int c = 0; c < NB; ++c)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[r][c][v] = 0.f;
  // two register batches of U steps: the next batch's loads are in flight while the
  // current one feeds the MFMAs
  bf16x8 wA[NB][U], xA[2][U], wB[NB][U], xB[2][U];
  auto load = [&](bf16x8 (&w)[NB][U], bf16x8 (&y)[2][U], int k) __attribute__((always_inline)) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
#pragma unroll
      for (int c = 0; c < NB; ++c) w[c][u] = *(const bf16x8*)(wp + c * wnb + k + 16 * u);
      y[0][u] = *(const bf16x8*)(x0 + k + 16 * u);
      y[1][u] = *(const bf16x8*)(x1 + k + 16 * u);
    }
  };
  auto mma = [&](const bf16x8 (&w)[NB][U], const bf16x8 (&y)[2][U])
      __attribute__((always_inline)) {
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int c = 0; c < NB; ++c)
#pragma unroll
        for (int r = 0; r < 2; ++r)
          acc[r][c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(y[r][u], w[c][u], acc[r][c], 0, 0, 0);
  };
  load(wA, xA, 0);
  for (int k = 0; k < kper; k += 32 * U) {
    const bool second = k + 16 * U < kper;
    if (second) load(wB, xB, k + 16 * U);
    mma(wA, xA);
    if (k + 32 * U < kper) load(wA, xA, k + 32 * U);
    if (second) mma(wB, xB);
  }
  // the four waves' partials are added in LDS in a fixed order, one 32-column block at a
  // time; accumulator element v of lane l is row 8 (v / 4) + 4 (l / 32) + v % 4, column
  // l % 32
#pragma unroll
  for (int c = 0; c < NB; ++c) {
    if (c > 0) __syncthreads();
#pragma unroll
    for (int v = 0; v < 16; ++v) {
      red[wave][0][v][lane] = acc[0][c][v];
      red[wave][1][v][lane] = acc[1][c][v];
    }
    __syncthreads();
    for (int e = tid; e < 2 * 16 * kWave; e += 256) {
      const int ln = e & (kWave - 1), v = (e / kWave) & 15, rb = e / (16 * kWave);
      const float sum = ((red[0][rb][v][ln] + red[1][rb][v][ln]) + red[2][rb][v][ln]) +
                        red[3][rb][v][ln];
      const int row = m0 + rb * 32 + 8 * (v >> 2) + 4 * (ln >> 5) + (v & 3);
      if (row < M) part[((size_t)split * M + row) * N + c0 + 32 * c + (ln & 31)] = sum;
    }
  }
}

// One wave per (tree node, head): blockIdx.x is the node (row = b * budget + i), and
// wave w of workgroup blockIdx.y takes head 4 blockIdx.y + w of the Hq query, Hkv key and
// Hkv value heads.  head_dim 128: lane l holds dims l and l + 64, the rotary pair.
__global__ __launch_bounds__(256) void qkv_rope_kernel(
    const float* __restrict__ part, int splits, int M, int budget, int Hq, int Hkv,
    const uint16_t* __restrict__ q_norm, const uint16_t* __restrict__ k_norm, double theta,
    float eps, const int64_t* __restrict__ off, const int32_t* __restrict__ ctxp,
    const int32_t* __restrict__ depthp, const int32_t* __restrict__ np_, int max_ctx,
    uint16_t* __restrict__ Q, uint16_t* __restrict__ Kc, uint16_t* __restrict__ Vc) {
  constexpr int HD = 128;
  const int row = blockIdx.x, b = row / budget, i = row - b * budget;
  const int n = min(max(np_[b], 0), budget);
  if (i >= n) return;
  const int ctx = min(max(ctxp[b], 0), max_ctx);
  const int pos = ctx + max(depthp[(size_t)b * budget + i], 0);
  const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
  const int hs = blockIdx.y * 4 + wave;
  if (hs >= Hq + 2 * Hkv) return;
  const int N = (Hq + 2 * Hkv) * HD;
  const size_t crow = (size_t)(off[b] + ctx + i) * Hkv;   // first head of the node's cache row
  // rotation of the pair (lane, lane + 64) at this position, from fp64 angles
  const double ang = (double)pos * pow(theta, -2.0 * (double)lane / (double)HD);
  double sd, cd;
  sincos(ang, &sd, &cd);
  const float sn = (float)sd, cs = (float)cd;
  {
    float x0 = 0.f, x1 = 0.f;
    for (int s = 0; s < splits; ++s) {
      const float* pr = part + ((size_t)s * M + row) * N + (size_t)hs * HD;
      x0 += pr[lane];
      x1 += pr[lane + 64];
    }
    if (hs >= Hq + Hkv) {             // value head: stored as projected
      const size_t o = (crow + (hs - Hq - Hkv)) * HD;
      Vc[o + lane] = f32_to_bf16(x0);
      Vc[o + lane + 64] = f32_to_bf16(x1);
      return;
    }
    float ss = x0 * x0 + x1 * x1;
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) ss += __shfl_xor(ss, m);
    const float r = 1.0f / sqrtf(ss * (1.0f / HD) + eps);
    const uint16_t* w = hs < Hq ? q_norm : k_norm;
    const float y0 = x0 * r * bf16_to_f32(w[lane]);
    const float y1 = x1 * r * bf16_to_f32(w[lane + 64]);
    const float z0 = y0 * cs - y1 * sn, z1 = y1 * cs + y0 * sn;
    uint16_t* dst = hs < Hq ? Q + ((size_t)row * Hq + hs) * HD : Kc + (crow + (hs - Hq)) * HD;
    dst[lane] = f32_to_bf16(z0);
    dst[lane + 64] = f32_to_bf16(z1);
  }
}

__global__ __launch_bounds__(256) void reduce_kernel(const float* __restrict__ part, int splits,
                                                     size_t total, uint16_t* __restrict__ Y) {
  const size_t e = ((size_t)blockIdx.x * 256 + threadIdx.x) * 4;
  if (e >= total) return;
  float4 s = *(const float4*)(part + e);
  for (int k = 1; k < splits; ++k) {
    const float4 t = *(const float4*)(part + (size_t)k * total + e);
    s.x += t.x;
    s.y += t.y;
    s.z += t.z;
    s.w += t.w;
  }
  const uint2 o = make_uint2((uint32_t)f32_to_bf16(s.x) | ((uint32_t)f32_to_bf16(s.y) << 16),
                             (uint32_t)f32_to_bf16(s.z) | ((uint32_t)f32_to_bf16(s.w) << 16));
  *(uint2*)(Y + e) = o;
}

}  // namespace

GemmPlan plan_gemm(int M, int N, int K) {
  GemmPlan p;
  // 64 columns per workgroup halve the re-reads of X against 32; N is a multiple of 64
  p.cols = N % 64 == 0 ? 64 : 32;
  const long long tiles = (long long)(N / p.cols) * ((M + 63) / 64);
  p.splits = 1;
  while (p.splits < 16 && tiles * p.splits < 256 && K % (2 * p.splits * 64) == 0) p.splits *= 2;
  const int steps = K / (p.splits * 4 * 16);
  p.unroll = p.cols == 64 ? 2 : 4;   // two batches in registers keep two waves per SIMD
  while (steps % p.unroll) p.unroll /= 2;
  return p;
}

hipError_t launch_gemm_bf16(const void* X, int M, int K, const void* w0, int n0, const void* w1,
                            int n1, const void* w2, int n2, const GemmPlan& p, float* part,
                            hipStream_t s) {
  const WSeg ws{(const uint16_t*)w0, (const uint16_t*)w1, (const uint16_t*)w2, n0, n0 + n1};
  const int N = n0 + n1 + n2;
  const dim3 grid((unsigned)(N / p.cols), (unsigned)p.splits, (unsigned)((M + 63) / 64));
  const uint16_t* x = (const uint16_t*)X;
#define TAPS_GEMM(UU, NBB) gemm_kernel<UU, NBB><<<grid, 256, 0, s>>>(x, M, K, ws, N, p.splits, part)
  if (p.cols == 64) {
    switch (p.unroll) {
      case 2: TAPS_GEMM(2, 2); break;
      default: TAPS_GEMM(1, 2); break;
    }
  } else {
    switch (p.unroll) {
      case 4: TAPS_GEMM(4, 1); break;
      case 2: TAPS_GEMM(2, 1); break;
      default: TAPS_GEMM(1, 1); break;
    }
  }
#undef TAPS_GEMM
  return hipGetLastError();
}

hipError_t launch_qkv_rope(const float* part, int splits, int batch, int budget, int Hq, int Hkv,
                           const void* q_norm, const void* k_norm, double theta, float eps,
                           const int64_t* off, const int32_t* ctx, const int32_t* depth,
                           const int32_t* n, int max_ctx, void* Q, void* Kc, void* Vc,
                           hipStream_t s) {
  const int M = batch * budget;
  const dim3 grid((unsigned)M, (unsigned)((Hq + 2 * Hkv + 3) / 4));
  qkv_rope_kernel<<<grid, 256, 0, s>>>(part, splits, M, budget, Hq, Hkv, (const uint16_t*)q_norm,
                                    (const uint16_t*)k_norm, theta, eps, off, ctx, depth, n,
                                    max_ctx, (uint16_t*)Q, (uint16_t*)Kc, (uint16_t*)Vc);
  return hipGetLastError();
}

hipError_t launch_reduce_bf16(const float* part, int splits, int M, int N, void* Y,
                              hipStream_t s) {
  const size_t total = (size_t)M * N;     // a multiple of 4 (N is a multiple of 64)
  const unsigned blocks = (unsigned)((total / 4 + 255) / 256);
  reduce_kernel<<<blocks, 256, 0, s>>>(part, splits, total, (uint16_t*)Y);
  return hipGetLastError();
}

}  // namespace taps
