// One attention layer of the target over the draft tree (the layer slice of the
// verification forward; Sec. 4.1 stage 3 and Sec. 4.3 run the target over the selected
// tree with tree attention), bf16 storage with fp32 accumulation.  Three kernels besides
// the tree attention of attn.hip:
//
//   gemm_kernel       Y_part = X W^T for a skinny X (the budget's nodes) and a large
//                     row-major weight [N][K]: HBM-bound on the weight, which is read once.
//                     A workgroup owns 64, 96 or 128 output columns, 64 rows and one split
//                     of K, planned so that the workgroups fill the 256 CUs in as few rounds
//                     as possible (one round of exactly 256 at the Qwen3-8B shapes).  The
//                     weight rows and X stream through a ring of LDS stages by direct loads
//                     (~60 KB of weight in flight per CU, which HBM's latency asks for);
//                     each of the four waves takes one 16-value k-step of every 64-value
//                     stage on v_mfma_f32_32x32x16_bf16, and the waves' partials are added in
//                     LDS in a fixed order.  Split partials (fp32) are added by the consumer.
//   qkv_rope_kernel   adds the projection's split partials, applies the per-head RMSNorm
//                     and the rotary embedding at position ctx + depth, and stores Q and the
//                     cache rows ctx + i of K and V in bf16.
//   reduce_kernel     adds the output projection's split partials and rounds to bf16.
#include "common.h"
#include "ldsload.h"

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

// Waits until at most c * PER vector-memory operations of this wave are outstanding, for a
// uniform c in [0, C] (s_waitcnt takes its count as an immediate).
template <int PER, int C>
__device__ inline void wait_later(int c) {
  if constexpr (C <= 0) {
    TAPS_WAIT_VMCNT(0);
  } else {
    if (c >= C) TAPS_WAIT_VMCNT(C * PER);
    else wait_later<PER, C - 1>(c);
  }
}

// XOR key of the 16-byte chunks of a 128-byte LDS row: 16 lanes reading the same logical
// chunk of 16 consecutive rows hit 16 distinct chunk positions of the 256-byte bank window
__device__ inline int row_swz(int r) { return (r >> 1) & 7; }

// Y_part[split] = X W^T over one split of K for 32 * NB output columns and 64 rows.
// Every global read is a direct load into a ring of D LDS stages; a stage is 64 values of K:
// the weight rows of the tile (32 * NB x 128 bytes) and the 64 X rows (64 x 128 bytes).
// Each 128-byte row keeps its 16-byte chunks XOR-permuted by row_swz.  Wave w takes the
// 16-value k-step w of every stage, so each wave holds a partial sum of the whole tile; the
// four partials are added in LDS in a fixed order at the end.
template <int NB, int D>
__global__ __launch_bounds__(256) void gemm_kernel(const uint16_t* __restrict__ X, int M, int K,
                                                   WSeg ws, int N, int splits,
                                                   float* __restrict__ part) {
  constexpr int WROWS = 32 * NB;     // weight rows (output columns) of the tile
  constexpr int WSLOT = WROWS * 128;
  constexpr int XSLOT = 64 * 128;
  constexpr int PER = NB + 2;        // direct loads per wave and stage (NB of W, 2 of X)
  constexpr int WPART = 2 * 16 * kWave;   // floats of one wave's partial of a column block
  static_assert(D * (WSLOT + XSLOT) >= NB * 4 * WPART * 4, "the reduction reuses the ring");
  static_assert((D - 2) * PER <= 63, "vmcnt counts at most 63 operations");
  __shared__ __attribute__((aligned(16))) unsigned char s_ring[D * (WSLOT + XSLOT)];
  asm volatile("" ::"s"(X), "s"(M), "s"(K), "s"(N), "s"(splits), "s"(part));
  const int c0 = blockIdx.x * WROWS, split = blockIdx.y, m0 = blockIdx.z * 64;
  const int tid = threadIdx.x, lane = tid & (kWave - 1);
  const int wave = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int l32 = lane & 31, hl = lane >> 5;
  const int Ks = K / splits, S = Ks / 64, kb = split * Ks;
  const uint32_t rowb = (uint32_t)K * 2;
  const int mrows = min(64, M - m0);

  // direct loads: wave-load g of a stage fills 1 KB = 8 rows (128 bytes each) of a slot;
  // lane i takes row 8g + i / 8, chunk position i % 8, i.e. global chunk
  // (i % 8) ^ row_swz(row).  Wave w issues W loads g = NB w .. NB w + NB - 1 (the tile's
  // weight rows 8g ..) and X loads g = 2w, 2w + 1.
  i32x4 wrs[NB];
  uint32_t woff[NB];
#pragma unroll
  for (int j = 0; j < NB; ++j) {
    const int g = NB * wave + j, gc = c0 + 8 * g;   // first output column of the 8 rows
    // the 8 rows lie in one weight array (its column count is a multiple of 8); the
    // resource covers exactly them
    const uint16_t* rows8 = gc < ws.end0   ? ws.w0 + (size_t)gc * K
                            : gc < ws.end1 ? ws.w1 + (size_t)(gc - ws.end0) * K
                                           : ws.w2 + (size_t)(gc - ws.end1) * K;
    wrs[j] = buffer_rsrc(rows8, 8u * rowb);
    const int r = 8 * g + (lane >> 3);
    woff[j] = (uint32_t)(lane >> 3) * rowb + (uint32_t)(kb + 8 * ((lane & 7) ^ row_swz(r))) * 2u;
  }
  const i32x4 xrs = buffer_rsrc(X + (size_t)m0 * K, (uint32_t)mrows * rowb);
  uint32_t xoff[2];
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int r = 8 * (2 * wave + j) + (lane >> 3);   // rows past M repeat row M - 1
    xoff[j] = (uint32_t)min(r, mrows - 1) * rowb +
              (uint32_t)(kb + 8 * ((lane & 7) ^ row_swz(r))) * 2u;
  }
  auto issue = [&](int slot, int st) __attribute__((always_inline)) {
    unsigned char* sw = s_ring + slot * WSLOT;
    unsigned char* sx = s_ring + D * WSLOT + slot * XSLOT;
#pragma unroll
    for (int j = 0; j < NB; ++j)
      load_lds16(wrs[j], sw + (NB * wave + j) * 1024, woff[j] + (uint32_t)st * 128u);
#pragma unroll
    for (int j = 0; j < 2; ++j)
      load_lds16(xrs, sx + (2 * wave + j) * 1024, xoff[j] + (uint32_t)st * 128u);
  };

  // MFMA operands: lane (l32, hl) reads 8 K values (chunk 2w + hl of the stage) of X row
  // l32 (+32) and of weight row l32 (+32 per column block)
  const int rdo = l32 * 128 + 16 * ((2 * wave + hl) ^ row_swz(l32));
  f32x16 acc[2][NB];
#pragma unroll
  for (int r = 0; r < 2; ++r)
#pragma unroll
    for (int c = 0; c < NB; ++c)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[r][c][v] = 0.f;
  auto compute = [&](int slot) __attribute__((always_inline)) {
    const unsigned char* sw = s_ring + slot * WSLOT + rdo;
    const unsigned char* sx = s_ring + D * WSLOT + slot * XSLOT + rdo;
    bf16x8 xa[2], wb[NB];
#pragma unroll
    for (int r = 0; r < 2; ++r) xa[r] = *(const bf16x8*)(sx + r * 32 * 128);
#pragma unroll
    for (int c = 0; c < NB; ++c) wb[c] = *(const bf16x8*)(sw + c * 32 * 128);
#pragma unroll
    for (int c = 0; c < NB; ++c)
#pragma unroll
      for (int r = 0; r < 2; ++r)
        acc[r][c] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(xa[r], wb[c], acc[r][c], 0, 0, 0);
  };

  // stages 0 .. D - 2 in flight first; at stage s, once its loads have landed (every
  // wave's: the barrier), slot (s - 1) % D is free and takes stage s + D - 1
  for (int s = 0; s < D - 1 && s < S; ++s) issue(s, s);
  for (int s0 = 0; s0 < S; s0 += D) {
#pragma unroll
    for (int i = 0; i < D; ++i) {
      const int s = s0 + i;
      if (s < S) {   // uniform; a guard, not an early exit, so that the loop unrolls fully
        // this wave's loads still allowed in flight: stages s + 1 .. min(S, s + D - 1) - 1
        const int later = min(S - 1 - s, D - 2);
        if (later == D - 2) TAPS_WAIT_VMCNT((D - 2) * PER);
        else wait_later<PER, D - 3>(later);
        TAPS_LDS_BARRIER();   // every wave's loads of stage s landed; slot (s - 1) % D is read
        if (s + D - 1 < S) issue((i + D - 1) % D, s + D - 1);
        compute(i);
      }
    }
  }
  TAPS_WAIT_VMCNT(0);
  __syncthreads();   // every wave is done with the ring

  // The four waves' partials of every column block go to LDS at once; then each thread
  // adds the four values of its outputs in a fixed order and stores the sums.  No barrier
  // follows the stores, so they all stay in flight together.  Accumulator element v of
  // lane l is row 8 (v / 4) + 4 (l / 32) + v % 4, column l % 32 of its 32 x 32 block.
  float* red = (float*)s_ring;   // [column block][wave][row block][v][lane]
#pragma unroll
  for (int c = 0; c < NB; ++c)
#pragma unroll
    for (int r = 0; r < 2; ++r)
#pragma unroll
      for (int v = 0; v < 16; ++v) red[(((c * 4 + wave) * 2 + r) * 16 + v) * kWave + lane] = acc[r][c][v];
  TAPS_LDS_BARRIER();
  // four consecutive columns of one row per thread and step: one 16-byte store each
  constexpr int Q4 = WPART / 4;
  const float4* red4 = (const float4*)s_ring;
#pragma unroll
  for (int k = 0; k < NB * Q4 / 256; ++k) {
    const int e4 = tid + 256 * k, c = e4 / Q4, w4 = e4 - c * Q4, e = 4 * w4;
    const int ln = e & (kWave - 1), v = (e / kWave) & 15, rb = e / (16 * kWave);
    const float4* q = red4 + c * 4 * Q4 + w4;
    const float4 a = q[0], b = q[Q4], d = q[2 * Q4], f = q[3 * Q4];
    const float4 sum = make_float4(((a.x + b.x) + d.x) + f.x, ((a.y + b.y) + d.y) + f.y,
                                   ((a.z + b.z) + d.z) + f.z, ((a.w + b.w) + d.w) + f.w);
    const int row = m0 + rb * 32 + 8 * (v >> 2) + 4 * (ln >> 5) + (v & 3);
    if (row < M) *(float4*)(part + ((size_t)split * M + row) * N + c0 + 32 * c + (ln & 31)) = sum;
  }
}

// One wave per (tree node, HPW heads): blockIdx.x is the node (row = b * budget + i), and
// wave w of workgroup blockIdx.y takes heads (4 blockIdx.y + w) HPW .. + HPW - 1 of the Hq
// query, Hkv key and Hkv value heads.  head_dim 128: lane l holds dims l and l + 64, the
// rotary pair; the wave's heads share the node's rotation, computed once.  SP = the
// projection's K splits: every load of the wave (the request's sizes, the node's depth and
// cache offset, and all SP partials of its heads) is issued before any of them is used, so
// the kernel waits for memory once.  In the paged kernel (PAGED), the node's cache row is
// logical row ctx + i of the request's pages (its page id needs ctx: one more round trip).
// Page ids outside the pool are clamped into it.
template <int SP, int HPW, bool PAGED>
__device__ __attribute__((always_inline)) inline void qkv_rope_body(
    const float* __restrict__ part, int M, int budget, int Hq, int Hkv,
    const uint16_t* __restrict__ q_norm, const uint16_t* __restrict__ k_norm, double theta,
    float eps, const int64_t* __restrict__ off, const int32_t* __restrict__ ctxp,
    const int32_t* __restrict__ depthp, const int32_t* __restrict__ np_, int max_ctx,
    uint16_t* __restrict__ Q, uint16_t* __restrict__ Kc, uint16_t* __restrict__ Vc, const PagedKV& pk) {
  constexpr int HD = 128;
  const int row = blockIdx.x, b = row / budget, i = row - b * budget;
  const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x / kWave;
  const int H = Hq + 2 * Hkv;
  const int h0 = (blockIdx.y * 4 + wave) * HPW;
  if (h0 >= H) return;
  const int N = H * HD;
  const int n_raw = np_[b], ctx_raw = ctxp[b], d_raw = depthp[(size_t)b * budget + i];
  int64_t kv0 = 0;
  if constexpr (!PAGED) kv0 = off[b];
  float p0[HPW][SP], p1[HPW][SP];
#pragma unroll
  for (int j = 0; j < HPW; ++j) {
    const int hs = min(h0 + j, H - 1);
#pragma unroll
    for (int s = 0; s < SP; ++s) {
      const float* pr = part + ((size_t)s * M + row) * N + (size_t)hs * HD;
      p0[j][s] = pr[lane];
      p1[j][s] = pr[lane + 64];
    }
  }
  const int n = min(max(n_raw, 0), budget);
  if (i >= n) return;
  const int ctx = min(max(ctx_raw, 0), max_ctx);
  const int pos = ctx + max(d_raw, 0);
  size_t crow;                                          // first head of the node's cache row
  if constexpr (PAGED) {
    const int L = ctx + i;
    int pg = pk.btab[(size_t)b * pk.max_pages + min(L >> pk.page_shift, pk.max_pages - 1)];
    pg = min(max(pg, 0), pk.num_pages - 1);
    crow = (((size_t)pg << pk.page_shift) | (size_t)(L & ((1 << pk.page_shift) - 1))) * Hkv;
  } else {
    crow = (size_t)(kv0 + ctx + i) * Hkv;
  }
  // rotation of the pair (lane, lane + 64) at this position, from fp64 angles
  float sn = 0.f, cs = 1.f;
  if (h0 < Hq + Hkv) {   // the wave holds a query or key head
    const double ang = (double)pos * pow(theta, -2.0 * (double)lane / (double)HD);
    double sd, cd;
    sincos(ang, &sd, &cd);
    sn = (float)sd;
    cs = (float)cd;
  }
#pragma unroll
  for (int j = 0; j < HPW; ++j) {
    const int hs = h0 + j;
    float x0 = 0.f, x1 = 0.f;
#pragma unroll
    for (int s = 0; s < SP; ++s) {   // the splits in order
      x0 += p0[j][s];
      x1 += p1[j][s];
    }
    if (hs >= Hq + Hkv && hs < H) {   // value head: stored as projected
      const size_t o = (crow + (hs - Hq - Hkv)) * HD;
      Vc[o + lane] = f32_to_bf16(x0);
      Vc[o + lane + 64] = f32_to_bf16(x1);
    } else if (hs < Hq + Hkv) {        // query or key head: RMSNorm and rotation
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
}

template <int SP, int HPW>
__global__ __launch_bounds__(256) void qkv_rope_kernel(
    const float* __restrict__ part, int M, int budget, int Hq, int Hkv,
    const uint16_t* __restrict__ q_norm, const uint16_t* __restrict__ k_norm, double theta,
    float eps, const int64_t* __restrict__ off, const int32_t* __restrict__ ctxp,
    const int32_t* __restrict__ depthp, const int32_t* __restrict__ np_, int max_ctx,
    uint16_t* __restrict__ Q, uint16_t* __restrict__ Kc, uint16_t* __restrict__ Vc) {
  qkv_rope_body<SP, HPW, false>(part, M, budget, Hq, Hkv, q_norm, k_norm, theta, eps, off, ctxp, depthp, np_, max_ctx, Q, Kc, Vc, PagedKV{nullptr, 0, 1, 5});
}

template <int SP, int HPW>
__global__ __launch_bounds__(256) void qkv_rope_paged_kernel(
    const float* __restrict__ part, int M, int budget, int Hq, int Hkv,
    const uint16_t* __restrict__ q_norm, const uint16_t* __restrict__ k_norm, double theta,
    float eps, const int64_t* __restrict__ off, const int32_t* __restrict__ ctxp,
    const int32_t* __restrict__ depthp, const int32_t* __restrict__ np_, int max_ctx,
    uint16_t* __restrict__ Q, uint16_t* __restrict__ Kc, uint16_t* __restrict__ Vc, PagedKV pk) {
  qkv_rope_body<SP, HPW, true>(part, M, budget, Hq, Hkv, q_norm, k_norm, theta, eps, off, ctxp, depthp, np_, max_ctx, Q, Kc, Vc, pk);
}

// Adds the output projection's SP split partials in order and rounds to bf16: four
// values per thread, all SP loads issued before the first addition.
template <int SP>
__global__ __launch_bounds__(256) void reduce_kernel(const float* __restrict__ part,
                                                     size_t total, uint16_t* __restrict__ Y) {
  const size_t e = ((size_t)blockIdx.x * 256 + threadIdx.x) * 4;
  if (e >= total) return;
  float4 t[SP];
#pragma unroll
  for (int k = 0; k < SP; ++k) t[k] = *(const float4*)(part + (size_t)k * total + e);
  float4 s = t[0];
#pragma unroll
  for (int k = 1; k < SP; ++k) {
    s.x += t[k].x;
    s.y += t[k].y;
    s.z += t[k].z;
    s.w += t[k].w;
  }
  const uint2 o = make_uint2((uint32_t)f32_to_bf16(s.x) | ((uint32_t)f32_to_bf16(s.y) << 16),
                             (uint32_t)f32_to_bf16(s.z) | ((uint32_t)f32_to_bf16(s.w) << 16));
  *(uint2*)(Y + e) = o;
}

}  // namespace

GemmPlan plan_gemm(int M, int N, int K) {
  // Candidates (64, 96 or 128 columns per workgroup; K splits 1 .. 16)
  // are ranked by how full their last round of workgroups leaves the 256 CUs (one
  // workgroup per CU: the ring takes most of the LDS), then by fewer rounds, then by fewer
  // splits (less partial traffic).  N is a multiple of 64 and K of 64, so 64 columns and
  // one split always qualify.
  const long long mt = (M + 63) / 64;
  GemmPlan best{1, 64};
  double best_fill = -1.0;
  long long best_rounds = 0;
  for (int nb = 2; nb <= 4; ++nb) {
    if (N % (32 * nb) != 0) continue;
    for (int sp = 1; sp <= 16 && K % (64 * sp) == 0; sp *= 2) {
      const long long wgs = (long long)(N / (32 * nb)) * sp * mt;
      const long long rounds = (wgs + 255) / 256;
      const double fill = (double)wgs / (double)(rounds * 256);
      const bool better =
          fill > best_fill + 1e-9 ||
          (fill > best_fill - 1e-9 &&
           (rounds < best_rounds || (rounds == best_rounds && sp < best.splits)));
      if (better) {
        best = GemmPlan{sp, 32 * nb};
        best_fill = fill;
        best_rounds = rounds;
      }
    }
  }
  return best;
}

hipError_t launch_gemm_bf16(const void* X, int M, int K, const void* w0, int n0, const void* w1,
                            int n1, const void* w2, int n2, const GemmPlan& p, float* part,
                            hipStream_t s) {
  const WSeg ws{(const uint16_t*)w0, (const uint16_t*)w1, (const uint16_t*)w2, n0, n0 + n1};
  const int N = n0 + n1 + n2;
  if (M <= 0) return hipSuccess;
  const dim3 grid((unsigned)(N / p.cols), (unsigned)p.splits, (unsigned)((M + 63) / 64));
  const uint16_t* x = (const uint16_t*)X;
  switch (p.cols) {   // ring depth: 120-144 KB of LDS
    case 64: gemm_kernel<2, 8><<<grid, 256, 0, s>>>(x, M, K, ws, N, p.splits, part); break;
    case 96: gemm_kernel<3, 6><<<grid, 256, 0, s>>>(x, M, K, ws, N, p.splits, part); break;
    case 128: gemm_kernel<4, 6><<<grid, 256, 0, s>>>(x, M, K, ws, N, p.splits, part); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_qkv_rope(const float* part, int splits, int batch, int budget, int Hq, int Hkv,
                           const void* q_norm, const void* k_norm, double theta, float eps,
                           const int64_t* off, const int32_t* ctx, const int32_t* depth,
                           const int32_t* n, int max_ctx, void* Q, void* Kc, void* Vc,
                           hipStream_t s, const PagedKV* pk) {

  const int M = batch * budget, H = Hq + 2 * Hkv;
  // four heads per wave once there are many (node, head) pairs: the fp64 rotation is then
  // computed once per four heads, and the grid still holds thousands of waves
  const int hpw = (long long)M * H > 8192 ? 4 : 1;
  const dim3 grid((unsigned)M, (unsigned)((H + 4 * hpw - 1) / (4 * hpw)));
#define TAPS_ROPE(SP, HPW)                                                                    \
  if (pk)                                                                                     \
    qkv_rope_paged_kernel<SP, HPW><<<grid, 256, 0, s>>>(                                      \
        part, M, budget, Hq, Hkv, (const uint16_t*)q_norm, (const uint16_t*)k_norm, theta, eps, \
        off, ctx, depth, n, max_ctx, (uint16_t*)Q, (uint16_t*)Kc, (uint16_t*)Vc, *pk);        \
  else                                                                                        \
    qkv_rope_kernel<SP, HPW><<<grid, 256, 0, s>>>(                                            \
        part, M, budget, Hq, Hkv, (const uint16_t*)q_norm, (const uint16_t*)k_norm, theta, eps, \
        off, ctx, depth, n, max_ctx, (uint16_t*)Q, (uint16_t*)Kc, (uint16_t*)Vc)
#define TAPS_ROPE_SP(SP)                \
  if (hpw == 4) {                       \
    TAPS_ROPE(SP, 4);                   \
  } else {                              \
    TAPS_ROPE(SP, 1);                   \
  }
  switch (splits) {   // the GEMM plan's split counts
    case 1: TAPS_ROPE_SP(1); break;
    case 2: TAPS_ROPE_SP(2); break;
    case 4: TAPS_ROPE_SP(4); break;
    case 8: TAPS_ROPE_SP(8); break;
    case 16: TAPS_ROPE_SP(16); break;
    default: return hipErrorInvalidValue;
  }
#undef TAPS_ROPE_SP
#undef TAPS_ROPE
  return hipGetLastError();
}

hipError_t launch_reduce_bf16(const float* part, int splits, int M, int N, void* Y,
                              hipStream_t s) {
  const size_t total = (size_t)M * N;     // a multiple of 4 (N is a multiple of 64)
  const unsigned blocks = (unsigned)((total / 4 + 255) / 256);
  switch (splits) {   // the GEMM plan's split counts
    case 1: reduce_kernel<1><<<blocks, 256, 0, s>>>(part, total, (uint16_t*)Y); break;
    case 2: reduce_kernel<2><<<blocks, 256, 0, s>>>(part, total, (uint16_t*)Y); break;
    case 4: reduce_kernel<4><<<blocks, 256, 0, s>>>(part, total, (uint16_t*)Y); break;
    case 8: reduce_kernel<8><<<blocks, 256, 0, s>>>(part, total, (uint16_t*)Y); break;
    case 16: reduce_kernel<16><<<blocks, 256, 0, s>>>(part, total, (uint16_t*)Y); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace taps
