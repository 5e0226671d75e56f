// KV commit of the accepted path (the round's state update after the acceptance walk;
// Sec. 1: each decoding round commits only one prefix path).
//
// The tree's K/V rows sit after the request's context, one per node.  The accepted path
// (root first, node indices strictly increasing because parents precede children) is
// gathered to the first rows after the context: row ctx + j <- row ctx + path[j].  As
// path[j] >= j, a target row can be the source row of an earlier path entry, never of a
// later one; every thread therefore reads all its source chunks before it writes any, and
// threads own disjoint 16-byte column chunks, so the in-place gather needs no barrier.
#include "common.h"

namespace taps {

namespace {

constexpr int kCommitThreads = 256;
constexpr int kMaxPath = TAPS_MAX_BLOCK + 1;   // root + one node per draft position
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Grid (column blocks, batch).  Thread t of block x owns 16-byte chunk x * 256 + t of the
// concatenated (K row, V row) of every path entry.  PAGED: Kc and Vc are page pools and
// request b's logical row r is page btab[b][r >> page_shift], slot r & (page_rows - 1);
// the gather is the same in logical rows, and the request's rows sit in distinct pages,
// so the in-place argument carries over.  Page ids outside the pool are clamped into it.
template <bool PAGED>
__device__ __attribute__((always_inline)) inline void commit_body(
    unsigned char* __restrict__ Kc, unsigned char* __restrict__ Vc,
    const int64_t* __restrict__ offp, const int32_t* __restrict__ ctxp,
    const int32_t* __restrict__ token, const int32_t* __restrict__ path,
    const int32_t* __restrict__ plen, const int32_t* __restrict__ bonus, int N, int D,
    int max_ctx, int row_chunks, int32_t* __restrict__ new_ctx, int32_t* __restrict__ committed,
    int32_t* __restrict__ n_committed, const PagedKV& pk) {
  const int b = blockIdx.y;
  const int c = blockIdx.x * kCommitThreads + threadIdx.x;
  const int32_t* pb = path + (size_t)b * (D + 1);
  // the committed path: root, then entries while they increase and stay below N
  const int m_in = min(max(plen[b], 1), D + 1);
  int m = 1, prev = 0;
  int src[kMaxPath];
  src[0] = 0;
#pragma unroll
  for (int j = 1; j < kMaxPath; ++j) {
    const int s = j < m_in ? pb[j] : -1;
    const bool ok = m == j && s > prev && s < N;
    src[j] = ok ? s : j;
    m = ok ? j + 1 : m;
    prev = ok ? s : prev;
  }
  const int ctx = min(max(ctxp[b], 0), max_ctx);

  if (c < 2 * row_chunks) {
    unsigned char* cache = c < row_chunks ? Kc : Vc;
    const int cc = c < row_chunks ? c : c - row_chunks;
    const size_t row_bytes = (size_t)row_chunks * 16;
    // this thread's chunk of tree row r (logical cache row ctx + r)
    unsigned char* col = nullptr;     // contiguous: the chunk of the request's first tree row
    if constexpr (!PAGED) col = cache + (size_t)(offp[b] + ctx) * row_bytes + (size_t)cc * 16;
    auto rowp = [&](int r) -> unsigned char* {
      if constexpr (PAGED) {
        const int L = ctx + r;
        int pg = pk.btab[(size_t)b * pk.max_pages + min(L >> pk.page_shift, pk.max_pages - 1)];
        pg = min(max(pg, 0), pk.num_pages - 1);
        const size_t phys = ((size_t)pg << pk.page_shift) | (size_t)(L & ((1 << pk.page_shift) - 1));
        return cache + phys * row_bytes + (size_t)cc * 16;
      } else {
        return col + (size_t)r * row_bytes;
      }
    };
    // entries past the path read the root's row (always the request's own) and are not
    // stored; all loads are issued before the first store
    u32x4 v[kMaxPath];
#pragma unroll
    for (int j = 1; j < kMaxPath; ++j) v[j] = *(const u32x4*)rowp(j < m ? src[j] : 0);
#pragma unroll
    for (int j = 1; j < kMaxPath; ++j)   // an entry at its own row stores what it read
      if (j < m) *(u32x4*)rowp(j) = v[j];
  }
  if (blockIdx.x == 0) {
    const int t = threadIdx.x;
    if (t <= D) {   // slot t: the token of path entry t + 1, then the bonus, then -1
      int32_t tok = -1;
      if (t + 1 < m) tok = token[(size_t)b * N + pb[t + 1]];
      else if (t + 1 == m) tok = bonus[b];
      committed[(size_t)b * (D + 1) + t] = tok;
    }
    if (t == 0) {
      new_ctx[b] = ctx + m;
      n_committed[b] = m;
    }
  }
}

// the contiguous cache keeps the kernel's original arguments; the paged one adds the table
__global__ __launch_bounds__(kCommitThreads) void commit_kernel(
    unsigned char* __restrict__ Kc, unsigned char* __restrict__ Vc,
    const int64_t* __restrict__ offp, const int32_t* __restrict__ ctxp,
    const int32_t* __restrict__ token, const int32_t* __restrict__ path,
    const int32_t* __restrict__ plen, const int32_t* __restrict__ bonus, int N, int D,
    int max_ctx, int row_chunks, int32_t* __restrict__ new_ctx, int32_t* __restrict__ committed,
    int32_t* __restrict__ n_committed) {
  commit_body<false>(Kc, Vc, offp, ctxp, token, path, plen, bonus, N, D, max_ctx, row_chunks, new_ctx, committed, n_committed, PagedKV{nullptr, 0, 1, 5});
}

__global__ __launch_bounds__(kCommitThreads) void commit_paged_kernel(
    unsigned char* __restrict__ Kc, unsigned char* __restrict__ Vc,
    const int64_t* __restrict__ offp, const int32_t* __restrict__ ctxp,
    const int32_t* __restrict__ token, const int32_t* __restrict__ path,
    const int32_t* __restrict__ plen, const int32_t* __restrict__ bonus, int N, int D,
    int max_ctx, int row_chunks, int32_t* __restrict__ new_ctx, int32_t* __restrict__ committed,
    int32_t* __restrict__ n_committed, PagedKV pk) {
  commit_body<true>(Kc, Vc, offp, ctxp, token, path, plen, bonus, N, D, max_ctx, row_chunks, new_ctx, committed, n_committed, pk);
}

}  // namespace

hipError_t launch_commit(void* K, void* V, const int64_t* off, const int32_t* ctx,
                         const int32_t* token, const int32_t* path, const int32_t* path_len,
                         const int32_t* bonus, int batch, int budget, int block, int Hkv,
                         int head_dim, int elem_bytes, int max_ctx, int32_t* new_ctx,
                         int32_t* committed, int32_t* n_committed, hipStream_t s,
                         const PagedKV* pk) {
  if (batch <= 0) return hipSuccess;
  const int row_chunks = Hkv * head_dim * elem_bytes / 16;
  const dim3 grid((unsigned)((2 * row_chunks + kCommitThreads - 1) / kCommitThreads),
                  (unsigned)batch);
  if (pk != nullptr)
    commit_paged_kernel<<<grid, kCommitThreads, 0, s>>>(
        (unsigned char*)K, (unsigned char*)V, off, ctx, token, path, path_len, bonus, budget,
        block, max_ctx, row_chunks, new_ctx, committed, n_committed, *pk);
  else
    commit_kernel<<<grid, kCommitThreads, 0, s>>>(
        (unsigned char*)K, (unsigned char*)V, off, ctx, token, path, path_len, bonus, budget,
        block, max_ctx, row_chunks, new_ctx, committed, n_committed);
  return hipGetLastError();
}

}  // namespace taps
