// C ABI entry points: host-side validation, workspace sizing and kernel dispatch.
#include <algorithm>
#include <cmath>
#include <cstdint>

#include "common.h"

using namespace taps;

namespace {

constexpr int kMaxChunks = 64;  // per-row chunk lists the selection kernel merges

bool finite(double x) { return std::isfinite(x); }

taps_status select_check(const taps_select_params* p) {
  if (!p) return TAPS_ERR_INVALID_ARG;
  if (p->batch < 0) return TAPS_ERR_INVALID_ARG;
  if (p->dtype != TAPS_BF16 && p->dtype != TAPS_FP32) return TAPS_ERR_INVALID_ARG;
  if (p->kind != TAPS_LOGITS && p->kind != TAPS_PROBS) return TAPS_ERR_INVALID_ARG;
  if (p->block < 1 || p->K < 1 || p->budget < 1 || p->vocab < 1) return TAPS_ERR_INVALID_ARG;
  if (p->block > TAPS_MAX_BLOCK || p->K > TAPS_MAX_K || p->budget > TAPS_MAX_BUDGET)
    return TAPS_ERR_UNSUPPORTED;
  if (p->K > p->vocab) return TAPS_ERR_INVALID_ARG;
  if (!finite(p->lambda1) || !(p->lambda1 > 0.0)) return TAPS_ERR_INVALID_ARG;
  if (!finite(p->lambda2)) return TAPS_ERR_INVALID_ARG;
  if (p->lambda2 < 0.0) return TAPS_ERR_UNSUPPORTED;
  if (std::isnan(p->tau)) return TAPS_ERR_INVALID_ARG;
  if (!finite(p->beta) || p->beta < 0.0) return TAPS_ERR_INVALID_ARG;
  if (p->kind == TAPS_PROBS && p->beta != 1.0) return TAPS_ERR_UNSUPPORTED;
  if (p->scorer != TAPS_SCORER_SIBLING && p->scorer != TAPS_SCORER_MARGINAL &&
      p->scorer != TAPS_SCORER_LEARNED)
    return TAPS_ERR_INVALID_ARG;
  if (p->scorer == TAPS_SCORER_MARGINAL && p->beta != 1.0) return TAPS_ERR_UNSUPPORTED;
  if (p->scorer == TAPS_SCORER_LEARNED) {
    if (p->kind != TAPS_LOGITS) return TAPS_ERR_UNSUPPORTED;
    if (p->block * p->K * p->K > kMaxLearnedEdges) return TAPS_ERR_UNSUPPORTED;
    const taps_scorer_mlp* w = p->mlp;
    if (!w || !w->emb || !w->W1 || !w->b1 || !w->w2 || !w->root_token)
      return TAPS_ERR_INVALID_ARG;
    if (w->emb_dim < 1 || w->hidden < 1) return TAPS_ERR_INVALID_ARG;
    if (w->emb_dim > 32 || w->hidden > 64) return TAPS_ERR_UNSUPPORTED;
    if (learned_chunk_units(p->block, p->K, w->emb_dim, w->hidden) < 1)
      return TAPS_ERR_UNSUPPORTED;
  }
  const int64_t rows = (int64_t)p->batch * p->block;
  if (rows > (int64_t)1 << 20) return TAPS_ERR_UNSUPPORTED;
  const TopkPlan plan = plan_topk(p->vocab, (int)rows > 0 ? (int)rows : 1, p->dtype);
  if (plan.chunks > kMaxChunks) return TAPS_ERR_UNSUPPORTED;
  return TAPS_OK;
}

bool needs_z(const taps_select_params* p) {
  return (p->scorer == TAPS_SCORER_MARGINAL && p->kind == TAPS_LOGITS) ||
         p->scorer == TAPS_SCORER_LEARNED;
}

taps_status attn_check(int32_t batch, int32_t budget, int32_t Hq, int32_t Hkv, int32_t hd,
                       int32_t max_ctx, int32_t dtype, float scale) {
  if (batch < 0 || budget < 1 || Hq < 1 || Hkv < 1 || max_ctx < 0) return TAPS_ERR_INVALID_ARG;
  if (budget > TAPS_MAX_BUDGET) return TAPS_ERR_UNSUPPORTED;
  if (Hq % Hkv != 0) return TAPS_ERR_INVALID_ARG;
  if (dtype != TAPS_BF16 && dtype != TAPS_FP32) return TAPS_ERR_INVALID_ARG;
  if (hd != 64 && hd != 128) return TAPS_ERR_UNSUPPORTED;
  if (!std::isfinite(scale) || !(scale > 0.f)) return TAPS_ERR_INVALID_ARG;
  if ((int64_t)max_ctx + budget > (int64_t)1 << 30) return TAPS_ERR_UNSUPPORTED;
  if ((int64_t)batch * Hkv > 65535 || (int64_t)budget * Hq / Hkv > (int64_t)1 << 20)
    return TAPS_ERR_UNSUPPORTED;
  // one request's queries must span < 2^31 bytes
  if ((int64_t)budget * Hq * hd * 2 >= ((int64_t)1 << 31)) return TAPS_ERR_UNSUPPORTED;
  // one split's K or V rows, with the kernel's look-ahead, must span < 2^31 bytes
  if ((int64_t)Hkv * hd * 2 * 6 * 64 >= ((int64_t)1 << 31)) return TAPS_ERR_UNSUPPORTED;
  return TAPS_OK;
}

struct LayerWs {
  size_t part, q, o, attn, total;
};

LayerWs layer_ws(int batch, int budget, int Hq, int Hkv, int hd, int hidden, int max_ctx,
                 int page_rows = 0) {
  const int M = batch * budget, Nqkv = (Hq + 2 * Hkv) * hd;
  const GemmPlan a = plan_gemm(M, Nqkv, hidden), o = plan_gemm(M, hidden, Hq * hd);
  auto al = [](size_t x) { return (x + 255) & ~(size_t)255; };
  LayerWs w;
  w.part = al(std::max((size_t)a.splits * M * Nqkv, (size_t)o.splits * M * hidden) * 4);
  w.q = al((size_t)M * Hq * hd * 2);
  w.o = w.q;
  w.attn = al(page_rows ? tree_verify_attn_paged_workspace_bytes(batch, budget, Hq, Hkv, hd,
                                                                 max_ctx, page_rows)
                        : tree_verify_attn_workspace_bytes(batch, budget, Hq, Hkv, hd, max_ctx,
                                                           TAPS_BF16));
  w.total = w.part + w.q + w.o + w.attn;
  return w;
}

taps_status layer_check(int32_t batch, int32_t budget, int32_t Hq, int32_t Hkv, int32_t hd,
                        int32_t hidden, int32_t max_ctx, float scale) {
  const taps_status st = attn_check(batch, budget, Hq, Hkv, hd, max_ctx, TAPS_BF16, scale);
  if (st != TAPS_OK) return st;
  if (hd != 128) return TAPS_ERR_UNSUPPORTED;
  if (hidden < 64 || hidden % 64 != 0) return TAPS_ERR_INVALID_ARG;
  if (hidden > 16384) return TAPS_ERR_UNSUPPORTED;
  if ((int64_t)batch * budget > ((int64_t)1 << 20)) return TAPS_ERR_UNSUPPORTED;
  return TAPS_OK;
}

}  // namespace

extern "C" {

const char* taps_status_string(int32_t s) {
  switch (s) {
    case TAPS_OK: return "TAPS_OK";
    case TAPS_ERR_INVALID_ARG: return "TAPS_ERR_INVALID_ARG";
    case TAPS_ERR_UNSUPPORTED: return "TAPS_ERR_UNSUPPORTED";
    case TAPS_ERR_WORKSPACE: return "TAPS_ERR_WORKSPACE";
    case TAPS_ERR_HIP: return "TAPS_ERR_HIP";
    default: return "TAPS_UNKNOWN_STATUS";
  }
}

double taps_spec_exp_host(double t) { return spec_exp_host(t); }

taps_status taps_select_validate(const taps_select_params* p) { return select_check(p); }

size_t taps_select_workspace_bytes(const taps_select_params* p) {
  if (select_check(p) != TAPS_OK || p->batch == 0) return 0;
  const int rows = p->batch * p->block;
  const TopkPlan plan = plan_topk(p->vocab, rows, p->dtype);
  const size_t cand = (size_t)rows * plan.chunks * p->K * sizeof(uint64_t);
  const size_t part = (size_t)rows * plan.chunks * kZSub * sizeof(int64_t);
  return cand + (needs_z(p) ? part : 0) + (p->scorer == TAPS_SCORER_LEARNED ? part : 0);
}

taps_status taps_select(const void* marginals, const taps_select_params* p, const taps_tree* out,
                        void* ws, size_t ws_bytes, hipStream_t stream) {
  const taps_status st = select_check(p);
  if (st != TAPS_OK) return st;
  if (p->batch == 0) return TAPS_OK;
  if (!marginals || !out || !out->parent || !out->token || !out->depth || !out->rank ||
      !out->q_reach || !out->n_nodes || !out->topk_idx)
    return TAPS_ERR_INVALID_ARG;
  if (((uintptr_t)marginals & 15) != 0) return TAPS_ERR_INVALID_ARG;
  const size_t need = taps_select_workspace_bytes(p);
  if (!ws || ws_bytes < need || ((uintptr_t)ws & 7) != 0) return TAPS_ERR_WORKSPACE;
  const int rows = p->batch * p->block;
  const TopkPlan plan = plan_topk(p->vocab, rows, p->dtype);
  if (launch_topk_chunks(marginals, p->dtype, rows, p->vocab, p->K, plan, (uint64_t*)ws,
                         stream) != hipSuccess)
    return TAPS_ERR_HIP;
  int64_t *zpart = nullptr, *spart = nullptr;
  if (needs_z(p)) {
    zpart = (int64_t*)((char*)ws + (size_t)rows * plan.chunks * p->K * sizeof(uint64_t));
    if (p->scorer == TAPS_SCORER_LEARNED) spart = zpart + (size_t)rows * plan.chunks * kZSub;
    if (launch_marginal_z(marginals, p->dtype, rows, p->vocab, p->K, plan, (const uint64_t*)ws,
                          zpart, spart, stream) != hipSuccess)
      return TAPS_ERR_HIP;
  }
  if (launch_select(marginals, *p, plan, (const uint64_t*)ws, zpart, spart, *out, stream) !=
      hipSuccess)
    return TAPS_ERR_HIP;
  return TAPS_OK;
}

taps_status tree_verify_attn_validate(int32_t batch, int32_t budget, int32_t Hq, int32_t Hkv,
                                      int32_t head_dim, int32_t max_ctx, int32_t dtype,
                                      float scale) {
  return attn_check(batch, budget, Hq, Hkv, head_dim, max_ctx, dtype, scale);
}

size_t tree_verify_attn_workspace_bytes(int32_t batch, int32_t budget, int32_t Hq, int32_t Hkv,
                                        int32_t head_dim, int32_t max_ctx, int32_t dtype) {
  if (attn_check(batch, budget, Hq, Hkv, head_dim, max_ctx, dtype, 1.0f) != TAPS_OK) return 0;
  if (dtype == TAPS_FP32 || batch == 0) return 0;
  const AttnPlan pl = plan_attn(batch, budget, Hq, Hkv, head_dim, max_ctx);
  return attn_ws_bytes(pl, batch, budget, Hq, Hkv, head_dim);
}

taps_status tree_verify_attn_timed(const void* Q_tree, const void* K_cache, const void* V_cache,
                                   const int64_t* kv_offset, const int32_t* ctx_len,
                                   const int32_t* tree_parent, const int32_t* n_nodes,
                                   int32_t batch, int32_t budget, int32_t Hq, int32_t Hkv,
                                   int32_t head_dim, int32_t max_ctx, int32_t dtype, float scale,
                                   void* O, void* ws, size_t ws_bytes, hipStream_t stream,
                                   hipEvent_t ev_begin, hipEvent_t ev_end) {
  const taps_status st = attn_check(batch, budget, Hq, Hkv, head_dim, max_ctx, dtype, scale);
  if (st != TAPS_OK) return st;
  if (batch == 0) return TAPS_OK;
  if (!Q_tree || !K_cache || !V_cache || !kv_offset || !ctx_len || !tree_parent || !n_nodes || !O)
    return TAPS_ERR_INVALID_ARG;
  const uintptr_t align_or = (uintptr_t)Q_tree | (uintptr_t)K_cache | (uintptr_t)V_cache | (uintptr_t)O;
  if ((align_or & 15) != 0) return TAPS_ERR_INVALID_ARG;
  if (dtype == TAPS_FP32) {
    return launch_attn_f32((const float*)Q_tree, (const float*)K_cache, (const float*)V_cache,
                           kv_offset, ctx_len, tree_parent, n_nodes, batch, budget, Hq, Hkv,
                           head_dim, max_ctx, scale, (float*)O, stream, ev_begin,
                           ev_end) == hipSuccess
               ? TAPS_OK
               : TAPS_ERR_HIP;
  }
  const size_t need = tree_verify_attn_workspace_bytes(batch, budget, Hq, Hkv, head_dim, max_ctx, dtype);
  if (!ws || ws_bytes < need || ((uintptr_t)ws & 15) != 0) return TAPS_ERR_WORKSPACE;
  const AttnPlan pl = plan_attn(batch, budget, Hq, Hkv, head_dim, max_ctx);
  return launch_attn_bf16(Q_tree, K_cache, V_cache, kv_offset, ctx_len, tree_parent, n_nodes,
                          batch, budget, Hq, Hkv, head_dim, max_ctx, scale, pl, O, ws, stream,
                          ev_begin, ev_end) == hipSuccess
             ? TAPS_OK
             : TAPS_ERR_HIP;
}

taps_status tree_verify_attn(const void* Q_tree, const void* K_cache, const void* V_cache,
                             const int64_t* kv_offset, const int32_t* ctx_len,
                             const int32_t* tree_parent, const int32_t* n_nodes, int32_t batch,
                             int32_t budget, int32_t Hq, int32_t Hkv, int32_t head_dim,
                             int32_t max_ctx, int32_t dtype, float scale, void* O, void* ws,
                             size_t ws_bytes, hipStream_t stream) {
  return tree_verify_attn_timed(Q_tree, K_cache, V_cache, kv_offset, ctx_len, tree_parent,
                                n_nodes, batch, budget, Hq, Hkv, head_dim, max_ctx, dtype, scale,
                                O, ws, ws_bytes, stream, nullptr, nullptr);
}

// log2 of a page size that is a power of two in [32, 4096], else -1
static int page_shift_of(int32_t page_rows) {
  if (page_rows < 32 || page_rows > 4096 || (page_rows & (page_rows - 1)) != 0) return -1;
  return __builtin_ctz((unsigned)page_rows);
}

static taps_status paged_check(int32_t batch, int32_t budget, int32_t Hq, int32_t Hkv,
                               int32_t head_dim, int32_t max_ctx, int32_t dtype, float scale,
                               int32_t page_rows) {
  const taps_status st = attn_check(batch, budget, Hq, Hkv, head_dim, max_ctx, dtype, scale);
  if (st != TAPS_OK) return st;
  if (page_shift_of(page_rows) < 0) return TAPS_ERR_INVALID_ARG;
  if (dtype != TAPS_BF16 || head_dim != 128) return TAPS_ERR_UNSUPPORTED;
  return TAPS_OK;
}

size_t tree_verify_attn_paged_workspace_bytes(int32_t batch, int32_t budget, int32_t Hq,
                                              int32_t Hkv, int32_t head_dim, int32_t max_ctx,
                                              int32_t page_rows) {
  if (paged_check(batch, budget, Hq, Hkv, head_dim, max_ctx, TAPS_BF16, 1.0f, page_rows) !=
          TAPS_OK ||
      batch == 0)
    return 0;
  const AttnPlan pl = plan_attn(batch, budget, Hq, Hkv, head_dim, max_ctx,
                                paged_max_split(page_shift_of(page_rows)));
  return attn_ws_bytes(pl, batch, budget, Hq, Hkv, head_dim);
}

taps_status tree_verify_attn_paged_timed(const void* Q_tree, const void* K_pages,
                                         const void* V_pages, int32_t num_pages,
                                         int32_t page_rows, const int32_t* block_table,
                                         int32_t max_pages, const int32_t* ctx_len,
                                         const int32_t* tree_parent, const int32_t* n_nodes,
                                         int32_t batch, int32_t budget, int32_t Hq, int32_t Hkv,
                                         int32_t head_dim, int32_t max_ctx, int32_t dtype,
                                         float scale, void* O, void* ws, size_t ws_bytes,
                                         hipStream_t stream, hipEvent_t ev_begin,
                                         hipEvent_t ev_end) {
  const taps_status st =
      paged_check(batch, budget, Hq, Hkv, head_dim, max_ctx, dtype, scale, page_rows);
  if (st != TAPS_OK) return st;
  if (num_pages < 1 || max_pages < 1) return TAPS_ERR_INVALID_ARG;
  // pool rows are addressed with 32-bit indices
  if ((int64_t)num_pages * page_rows > (int64_t)UINT32_MAX) return TAPS_ERR_UNSUPPORTED;
  // every logical row a request may own (its context and its nodes) has a table entry
  if ((int64_t)max_pages * page_rows < (int64_t)max_ctx + budget) return TAPS_ERR_INVALID_ARG;
  if (batch == 0) return TAPS_OK;
  if (!Q_tree || !K_pages || !V_pages || !block_table || !ctx_len || !tree_parent || !n_nodes ||
      !O)
    return TAPS_ERR_INVALID_ARG;
  const uintptr_t align_or =
      (uintptr_t)Q_tree | (uintptr_t)K_pages | (uintptr_t)V_pages | (uintptr_t)O;
  if ((align_or & 15) != 0 || ((uintptr_t)block_table & 3) != 0) return TAPS_ERR_INVALID_ARG;
  const size_t need = tree_verify_attn_paged_workspace_bytes(batch, budget, Hq, Hkv, head_dim,
                                                             max_ctx, page_rows);
  if (!ws || ws_bytes < need || ((uintptr_t)ws & 15) != 0) return TAPS_ERR_WORKSPACE;
  const int shift = page_shift_of(page_rows);
  const AttnPlan pl = plan_attn(batch, budget, Hq, Hkv, head_dim, max_ctx, paged_max_split(shift));
  return launch_attn_bf16_paged(Q_tree, K_pages, V_pages, block_table, max_pages, num_pages,
                                shift, ctx_len, tree_parent, n_nodes, batch, budget, Hq, Hkv,
                                max_ctx, scale, pl, O, ws, stream, ev_begin,
                                ev_end) == hipSuccess
             ? TAPS_OK
             : TAPS_ERR_HIP;
}

taps_status tree_verify_attn_paged(const void* Q_tree, const void* K_pages, const void* V_pages,
                                   int32_t num_pages, int32_t page_rows,
                                   const int32_t* block_table, int32_t max_pages,
                                   const int32_t* ctx_len, const int32_t* tree_parent,
                                   const int32_t* n_nodes, int32_t batch, int32_t budget,
                                   int32_t Hq, int32_t Hkv, int32_t head_dim, int32_t max_ctx,
                                   int32_t dtype, float scale, void* O, void* ws,
                                   size_t ws_bytes, hipStream_t stream) {
  return tree_verify_attn_paged_timed(Q_tree, K_pages, V_pages, num_pages, page_rows,
                                      block_table, max_pages, ctx_len, tree_parent, n_nodes,
                                      batch, budget, Hq, Hkv, head_dim, max_ctx, dtype, scale, O,
                                      ws, ws_bytes, stream, nullptr, nullptr);
}

taps_status accept_walk(const taps_tree* tree, int32_t batch, int32_t budget, int32_t block,
                        const int32_t* target_tokens, int32_t* path, int32_t* path_len,
                        int32_t* bonus, hipStream_t stream) {
  if (batch < 0 || budget < 1 || block < 1) return TAPS_ERR_INVALID_ARG;
  if (budget > TAPS_MAX_BUDGET || block > TAPS_MAX_BLOCK) return TAPS_ERR_UNSUPPORTED;
  if (batch == 0) return TAPS_OK;
  if (!tree || !tree->parent || !tree->token || !tree->n_nodes || !target_tokens || !path ||
      !path_len || !bonus)
    return TAPS_ERR_INVALID_ARG;
  return launch_walk(*tree, batch, budget, block, target_tokens, path, path_len, bonus, stream) ==
                 hipSuccess
             ? TAPS_OK
             : TAPS_ERR_HIP;
}

static taps_status commit_check(int32_t batch, int32_t budget, int32_t block, int32_t Hkv,
                                int32_t head_dim, int32_t max_ctx, int32_t dtype) {
  if (batch < 0 || budget < 1 || block < 1 || Hkv < 1 || max_ctx < 0)
    return TAPS_ERR_INVALID_ARG;
  if (budget > TAPS_MAX_BUDGET || block > TAPS_MAX_BLOCK) return TAPS_ERR_UNSUPPORTED;
  if (head_dim != 64 && head_dim != 128) return TAPS_ERR_UNSUPPORTED;
  if (dtype != TAPS_BF16 && dtype != TAPS_FP32) return TAPS_ERR_INVALID_ARG;
  if ((int64_t)Hkv * head_dim * 4 > ((int64_t)1 << 24)) return TAPS_ERR_UNSUPPORTED;
  if ((int64_t)max_ctx + budget > (int64_t)1 << 30) return TAPS_ERR_UNSUPPORTED;
  if (batch > 65535) return TAPS_ERR_UNSUPPORTED;
  return TAPS_OK;
}

taps_status kv_commit_paged(void* K_pages, void* V_pages, int32_t num_pages, int32_t page_rows,
                            const int32_t* block_table, int32_t max_pages,
                            const int32_t* ctx_len, const taps_tree* tree, const int32_t* path,
                            const int32_t* path_len, const int32_t* bonus, int32_t batch,
                            int32_t budget, int32_t block, int32_t Hkv, int32_t head_dim,
                            int32_t max_ctx, int32_t dtype, int32_t* new_ctx_len,
                            int32_t* committed, int32_t* n_committed, hipStream_t stream) {
  const taps_status st = commit_check(batch, budget, block, Hkv, head_dim, max_ctx, dtype);
  if (st != TAPS_OK) return st;
  const int shift = page_shift_of(page_rows);
  if (shift < 0 || num_pages < 1 || max_pages < 1) return TAPS_ERR_INVALID_ARG;
  if ((int64_t)max_pages * page_rows < (int64_t)max_ctx + budget) return TAPS_ERR_INVALID_ARG;
  if (batch == 0) return TAPS_OK;
  if (!K_pages || !V_pages || !block_table || !ctx_len || !tree || !tree->token || !path ||
      !path_len || !bonus || !new_ctx_len || !committed || !n_committed)
    return TAPS_ERR_INVALID_ARG;
  if ((((uintptr_t)K_pages | (uintptr_t)V_pages) & 15) != 0 || ((uintptr_t)block_table & 3) != 0)
    return TAPS_ERR_INVALID_ARG;
  if ((const void*)new_ctx_len == (const void*)ctx_len) return TAPS_ERR_INVALID_ARG;
  const PagedKV pk{block_table, max_pages, num_pages, shift};
  return launch_commit(K_pages, V_pages, nullptr, ctx_len, tree->token, path, path_len, bonus,
                       batch, budget, block, Hkv, head_dim, dtype == TAPS_BF16 ? 2 : 4, max_ctx,
                       new_ctx_len, committed, n_committed, stream, &pk) == hipSuccess
             ? TAPS_OK
             : TAPS_ERR_HIP;
}

taps_status kv_commit(void* K_cache, void* V_cache, const int64_t* kv_offset,
                      const int32_t* ctx_len, const taps_tree* tree, const int32_t* path,
                      const int32_t* path_len, const int32_t* bonus, int32_t batch,
                      int32_t budget, int32_t block, int32_t Hkv, int32_t head_dim,
                      int32_t max_ctx, int32_t dtype, int32_t* new_ctx_len, int32_t* committed,
                      int32_t* n_committed, hipStream_t stream) {
  if (batch < 0 || budget < 1 || block < 1 || Hkv < 1 || max_ctx < 0)
    return TAPS_ERR_INVALID_ARG;
  if (budget > TAPS_MAX_BUDGET || block > TAPS_MAX_BLOCK) return TAPS_ERR_UNSUPPORTED;
  if (head_dim != 64 && head_dim != 128) return TAPS_ERR_UNSUPPORTED;
  if (dtype != TAPS_BF16 && dtype != TAPS_FP32) return TAPS_ERR_INVALID_ARG;
  if ((int64_t)Hkv * head_dim * 4 > ((int64_t)1 << 24)) return TAPS_ERR_UNSUPPORTED;
  if ((int64_t)max_ctx + budget > (int64_t)1 << 30) return TAPS_ERR_UNSUPPORTED;
  if (batch == 0) return TAPS_OK;
  if (!K_cache || !V_cache || !kv_offset || !ctx_len || !tree || !tree->token || !path ||
      !path_len || !bonus || !new_ctx_len || !committed || !n_committed)
    return TAPS_ERR_INVALID_ARG;
  if ((((uintptr_t)K_cache | (uintptr_t)V_cache) & 15) != 0) return TAPS_ERR_INVALID_ARG;
  if ((const void*)new_ctx_len == (const void*)ctx_len) return TAPS_ERR_INVALID_ARG;
  if (batch > 65535) return TAPS_ERR_UNSUPPORTED;
  const int elem = dtype == TAPS_BF16 ? 2 : 4;
  return launch_commit(K_cache, V_cache, kv_offset, ctx_len, tree->token, path, path_len, bonus,
                       batch, budget, block, Hkv, head_dim, elem, max_ctx, new_ctx_len,
                       committed, n_committed, stream) == hipSuccess
             ? TAPS_OK
             : TAPS_ERR_HIP;
}

size_t verify_layer_workspace_bytes(int32_t batch, int32_t budget, int32_t Hq, int32_t Hkv,
                                    int32_t head_dim, int32_t hidden, int32_t max_ctx) {
  if (layer_check(batch, budget, Hq, Hkv, head_dim, hidden, max_ctx, 1.0f) != TAPS_OK ||
      batch == 0)
    return 0;
  return layer_ws(batch, budget, Hq, Hkv, head_dim, hidden, max_ctx).total;
}

// The layer over a contiguous cache (pk == nullptr) or a paged one (C20)
static taps_status layer_run(const void* X, const taps_layer_weights* w, void* K_cache,
                             void* V_cache, const int64_t* kv_offset, const int32_t* ctx_len,
                             const taps_tree* tree, int32_t batch, int32_t budget, int32_t Hq,
                             int32_t Hkv, int32_t head_dim, int32_t max_ctx, float scale,
                             void* Y, void* ws, size_t ws_bytes, hipStream_t stream,
                             const PagedKV* pk, int32_t page_rows) {
  if (!w) return TAPS_ERR_INVALID_ARG;
  const taps_status st = layer_check(batch, budget, Hq, Hkv, head_dim, w->hidden, max_ctx, scale);
  if (st != TAPS_OK) return st;
  if (!std::isfinite(w->rope_theta) || !(w->rope_theta > 1.0)) return TAPS_ERR_INVALID_ARG;
  if (!std::isfinite(w->norm_eps) || w->norm_eps < 0.f) return TAPS_ERR_INVALID_ARG;
  if (batch == 0) return TAPS_OK;
  if (!X || !Y || !K_cache || !V_cache || (!kv_offset && !pk) || !ctx_len || !tree ||
      !tree->parent ||
      !tree->depth || !tree->n_nodes || !w->Wq || !w->Wk || !w->Wv || !w->Wo || !w->q_norm ||
      !w->k_norm)
    return TAPS_ERR_INVALID_ARG;
  const uintptr_t a16 = (uintptr_t)X | (uintptr_t)Y | (uintptr_t)K_cache | (uintptr_t)V_cache |
                        (uintptr_t)w->Wq | (uintptr_t)w->Wk | (uintptr_t)w->Wv | (uintptr_t)w->Wo;
  if ((a16 & 15) != 0 || (((uintptr_t)w->q_norm | (uintptr_t)w->k_norm) & 1) != 0)
    return TAPS_ERR_INVALID_ARG;
  const int hidden = w->hidden;
  const LayerWs L = layer_ws(batch, budget, Hq, Hkv, head_dim, hidden, max_ctx, pk ? page_rows : 0);
  if (!ws || ws_bytes < L.total || ((uintptr_t)ws & 255) != 0) return TAPS_ERR_WORKSPACE;
  const int M = batch * budget, Nq = Hq * head_dim, Nk = Hkv * head_dim;
  float* part = (float*)ws;
  char* Q = (char*)ws + L.part;
  char* O = Q + L.q;
  char* aws = O + L.o;
  const GemmPlan a = plan_gemm(M, Nq + 2 * Nk, hidden);
  if (launch_gemm_bf16(X, M, hidden, w->Wq, Nq, w->Wk, Nk, w->Wv, Nk, a, part, stream) !=
      hipSuccess)
    return TAPS_ERR_HIP;
  if (launch_qkv_rope(part, a.splits, batch, budget, Hq, Hkv, w->q_norm, w->k_norm,
                      w->rope_theta, w->norm_eps, kv_offset, ctx_len, tree->depth,
                      tree->n_nodes, max_ctx, Q, K_cache, V_cache, stream, pk) != hipSuccess)
    return TAPS_ERR_HIP;
  if (pk) {
    const AttnPlan pl = plan_attn(batch, budget, Hq, Hkv, head_dim, max_ctx,
                                  paged_max_split(pk->page_shift));
    if (launch_attn_bf16_paged(Q, K_cache, V_cache, pk->btab, pk->max_pages, pk->num_pages,
                               pk->page_shift, ctx_len, tree->parent, tree->n_nodes, batch,
                               budget, Hq, Hkv, max_ctx, scale, pl, O, aws, stream) !=
        hipSuccess)
      return TAPS_ERR_HIP;
  } else {
    const AttnPlan pl = plan_attn(batch, budget, Hq, Hkv, head_dim, max_ctx);
    if (launch_attn_bf16(Q, K_cache, V_cache, kv_offset, ctx_len, tree->parent, tree->n_nodes,
                         batch, budget, Hq, Hkv, head_dim, max_ctx, scale, pl, O, aws,
                         stream) != hipSuccess)
      return TAPS_ERR_HIP;
  }
  const GemmPlan o = plan_gemm(M, hidden, Nq);
  if (launch_gemm_bf16(O, M, Nq, w->Wo, hidden, nullptr, 0, nullptr, 0, o, part, stream) !=
      hipSuccess)
    return TAPS_ERR_HIP;
  return launch_reduce_bf16(part, o.splits, M, hidden, Y, stream) == hipSuccess ? TAPS_OK
                                                                                : TAPS_ERR_HIP;
}

taps_status verify_layer(const void* X, const taps_layer_weights* w, void* K_cache,
                         void* V_cache, const int64_t* kv_offset, const int32_t* ctx_len,
                         const taps_tree* tree, int32_t batch, int32_t budget, int32_t Hq,
                         int32_t Hkv, int32_t head_dim, int32_t max_ctx, float scale, void* Y,
                         void* ws, size_t ws_bytes, hipStream_t stream) {
  return layer_run(X, w, K_cache, V_cache, kv_offset, ctx_len, tree, batch, budget, Hq, Hkv,
                   head_dim, max_ctx, scale, Y, ws, ws_bytes, stream, nullptr, 0);
}

size_t verify_layer_paged_workspace_bytes(int32_t batch, int32_t budget, int32_t Hq,
                                          int32_t Hkv, int32_t head_dim, int32_t hidden,
                                          int32_t max_ctx, int32_t page_rows) {
  if (layer_check(batch, budget, Hq, Hkv, head_dim, hidden, max_ctx, 1.0f) != TAPS_OK ||
      page_shift_of(page_rows) < 0 || batch == 0)
    return 0;
  return layer_ws(batch, budget, Hq, Hkv, head_dim, hidden, max_ctx, page_rows).total;
}

taps_status verify_layer_paged(const void* X, const taps_layer_weights* w, void* K_pages,
                               void* V_pages, int32_t num_pages, int32_t page_rows,
                               const int32_t* block_table, int32_t max_pages,
                               const int32_t* ctx_len, const taps_tree* tree, int32_t batch,
                               int32_t budget, int32_t Hq, int32_t Hkv, int32_t head_dim,
                               int32_t max_ctx, float scale, void* Y, void* ws, size_t ws_bytes,
                               hipStream_t stream) {
  const int shift = page_shift_of(page_rows);
  if (shift < 0 || num_pages < 1 || max_pages < 1) return TAPS_ERR_INVALID_ARG;
  if ((int64_t)max_pages * page_rows < (int64_t)max_ctx + budget) return TAPS_ERR_INVALID_ARG;
  if ((int64_t)num_pages * page_rows > (int64_t)UINT32_MAX) return TAPS_ERR_UNSUPPORTED;
  if (batch > 0 && (!block_table || ((uintptr_t)block_table & 3) != 0))
    return TAPS_ERR_INVALID_ARG;
  const PagedKV pk{block_table, max_pages, num_pages, shift};
  return layer_run(X, w, K_pages, V_pages, nullptr, ctx_len, tree, batch, budget, Hq, Hkv,
                   head_dim, max_ctx, scale, Y, ws, ws_bytes, stream, &pk, page_rows);
}

}  // extern "C"
