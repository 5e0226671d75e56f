// Internal declarations shared by the HIP translation units of libtaps.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>
#include "../../include/taps.h"

namespace taps {

constexpr int kWave = 64;

// ----------------------------------------------------------------------------------
// Order-preserving keys for marginal values.  A larger key ranks earlier: value
// descending with -0 == +0 and every NaN below -inf.  The 64-bit candidate key packs
// (value key << 32) | ~index, so equal values rank by ascending vocabulary index and
// every key is unique.
__host__ __device__ inline uint32_t value_key(uint32_t bits) {
  if ((bits & 0x7FFFFFFFu) > 0x7F800000u) return 0u;  // NaN
  if (bits == 0x80000000u) bits = 0u;                 // -0 -> +0
  return (bits & 0x80000000u) ? ~bits : (bits | 0x80000000u);
}
__host__ __device__ inline uint64_t cand_key(uint32_t vkey, uint32_t idx) {
  return ((uint64_t)vkey << 32) | (uint64_t)(0xFFFFFFFFu - idx);
}
__host__ __device__ inline uint32_t cand_index(uint64_t key) {
  return 0xFFFFFFFFu - (uint32_t)(key & 0xFFFFFFFFu);
}

// ----------------------------------------------------------------------------------
// Host launchers (each returns hipGetLastError() of its launch).
struct TopkPlan {
  int chunk_len;   // elements per chunk (multiple of 1024)
  int chunks;      // chunks per row
  int per_thread;  // elements per thread (chunk_len / 256)
};
TopkPlan plan_topk(int vocab, int rows, int dtype);

hipError_t launch_topk_chunks(const void* marg, int dtype, int rows, int vocab, int K,
                              const TopkPlan& plan, uint64_t* cand, hipStream_t s);

hipError_t launch_select(const void* marg, const taps_select_params& p, const TopkPlan& plan,
                         const uint64_t* cand, const int64_t* zpart, const int64_t* spart,
                         const taps_tree& out, hipStream_t s);

// Integer partials of a row's full-vocabulary sums per top-K chunk (one workgroup each)
constexpr int kZSub = 4;

// Largest q_cond table D*K*K of the learned scorer (fp64, in dynamic LDS)
constexpr int kMaxLearnedEdges = 7168;

// Hidden units per chunk of the learned scorer's working set (0: it does not fit)
int learned_chunk_units(int D, int K, int emb_dim, int hidden);

hipError_t launch_marginal_z(const void* marg, int dtype, int rows, int vocab, int K,
                             const TopkPlan& plan, const uint64_t* cand, int64_t* zpart,
                             int64_t* spart, hipStream_t s);

struct AttnPlan {
  int qb;          // 32-row query blocks per wave (1 or 2)
  int wk;          // key groups per workgroup (1 or 2): 256 * wk threads
  int mtile;       // query rows per workgroup (4 waves)
  int mtiles;      // workgroups along the budget*G query rows of one KV head
  int split_len;   // keys per split (multiple of 64); 0 when ragged
  int splits;      // splits along max_ctx + budget keys; 1 when ragged
  // Ragged work list (several requests, head_dim 128): the kernel sizes the splits from the
  // requests' actual keys so that the batch makes about target_pairs (request, KV head,
  // split) pairs; at most pairs_max; split lengths at most lcap keys
  int ragged;
  int target_pairs;
  int pairs_max;
  int lcap;
};
// Paged KV cache: block table [batch][max_pages] of page ids into pools of num_pages pages
// of 2^page_shift rows
struct PagedKV {
  const int32_t* btab;
  int max_pages, num_pages, page_shift;
};

// max_len > 0 caps the split length (a multiple of 32): paged calls, whose splits may span
// at most a fixed number of pages
AttnPlan plan_attn(int batch, int budget, int Hq, int Hkv, int head_dim, int max_ctx,
                   int max_len = 0);
size_t attn_ws_bytes(const AttnPlan& pl, int batch, int budget, int Hq, int Hkv, int head_dim);

hipError_t launch_attn_bf16(const void* Q, const void* K, const void* V, const int64_t* off,
                            const int32_t* ctx, const int32_t* parent, const int32_t* n,
                            int batch, int budget, int Hq, int Hkv, int head_dim, int max_ctx,
                            float scale, const AttnPlan& pl, void* O, void* ws, hipStream_t s,
                            hipEvent_t ev_begin = nullptr, hipEvent_t ev_end = nullptr);

// Paged K/V (head_dim 128, bf16): pools [num_pages][2^page_shift][Hkv][128], request b's
// logical row r at page block_table[b * max_pages + (r >> page_shift)]
hipError_t launch_attn_bf16_paged(const void* Q, const void* K_pages, const void* V_pages,
                                  const int32_t* block_table, int max_pages, int num_pages,
                                  int page_shift, const int32_t* ctx, const int32_t* parent,
                                  const int32_t* n, int batch, int budget, int Hq, int Hkv,
                                  int max_ctx, float scale, const AttnPlan& pl, void* O,
                                  void* ws, hipStream_t s, hipEvent_t ev_begin = nullptr,
                                  hipEvent_t ev_end = nullptr);
// longest split a paged call may take: its page ids must fit the kernel's table
int paged_max_split(int page_shift);

hipError_t launch_attn_f32(const float* Q, const float* K, const float* V, const int64_t* off,
                           const int32_t* ctx, const int32_t* parent, const int32_t* n,
                           int batch, int budget, int Hq, int Hkv, int head_dim, int max_ctx,
                           float scale, float* O, hipStream_t s, hipEvent_t ev_begin = nullptr,
                           hipEvent_t ev_end = nullptr);

hipError_t launch_walk(const taps_tree& t, int batch, int budget, int block,
                       const int32_t* target, int32_t* path, int32_t* path_len, int32_t* bonus,
                       hipStream_t s);

// pk != nullptr: K and V are page pools addressed through pk's block table (off unused)
hipError_t launch_commit(void* K, void* V, const int64_t* off, const int32_t* ctx,
                         const int32_t* token, const int32_t* path, const int32_t* path_len,
                         const int32_t* bonus, int batch, int budget, int block, int Hkv,
                         int head_dim, int elem_bytes, int max_ctx, int32_t* new_ctx,
                         int32_t* committed, int32_t* n_committed, hipStream_t s,
                         const PagedKV* pk = nullptr);

// Layer slice: split-K skinny GEMM (fp32 partials [splits][M][N]), the projection
// epilogue (RMSNorm, rotary positions, bf16 Q and cache rows) and the output reduction
struct GemmPlan {
  int splits;   // K splits (partials), each a multiple of 64 K values
  int cols;     // output columns per workgroup (64, 96 or 128)
};
GemmPlan plan_gemm(int M, int N, int K);
hipError_t launch_gemm_bf16(const void* X, int M, int K, const void* w0, int n0, const void* w1,
                            int n1, const void* w2, int n2, const GemmPlan& p, float* part,
                            hipStream_t s);
hipError_t launch_qkv_rope(const float* part, int splits, int batch, int budget, int Hq, int Hkv,
                           const void* q_norm, const void* k_norm, double theta, float eps,
                           const int64_t* off, const int32_t* ctx, const int32_t* depth,
                           const int32_t* n, int max_ctx, void* Q, void* Kc, void* Vc,
                           hipStream_t s, const PagedKV* pk = nullptr);
hipError_t launch_reduce_bf16(const float* part, int splits, int M, int N, void* Y,
                              hipStream_t s);

double spec_exp_host(double t);

}  // namespace taps
