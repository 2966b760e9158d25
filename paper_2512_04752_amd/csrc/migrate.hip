// KV transfer buffer for sample migration (RLHFSpec Section 6.2, "Two-stage
// Sample Migration", phases 1 and 3): the K/V of chosen token ranges of
// several samples is copied out of the KV pool into one contiguous buffer, so
// that a migration is a single copy, and parsed back into another pool.
//
// Buffer order (the paper's model -> layer -> sample hierarchy; the LLM is the
// only model here):
//   [layer][K=0,V=1][sample j in call order][kv_head][token t in [begin_j, end_j)][head_dim]
// so every (layer, K/V, sample, head) run of count_j * head_dim values is
// contiguous both in the buffer and in the pool (where one (layer, K/V, head)
// of a sample is [capacity][head_dim]).
//
// One work-group copies one chunk of kChunk 16-byte units of one such run:
// the grid is ordered [layer, K/V][sample][head][chunk], the work-group
// decodes its run once (a binary search over the samples' work-group prefix),
// then streams the chunk with every load of a thread in flight before its
// stores.  The copy is HBM-bound: 2 bytes moved per byte of K/V.
#include "common.h"

namespace spec {

namespace {

constexpr int kChunk = 4096;               // 16-byte units per work-group (64 KB)
constexpr int kPer = kChunk / 256;         // units per thread

template <bool TO_BUFFER>
__global__ __launch_bounds__(256) void kv_transfer_kernel(const MigrateInfo* info, int n,
                                                          int64_t wg_per_slab, int tok_total,
                                                          bf16* pool, bf16* buf, int n_kv_heads,
                                                          int head_dim) {
  const int64_t wg = blockIdx.x;
  const int lk = (int)(wg / wg_per_slab);            // layer * 2 + (K=0, V=1)
  const int64_t rem = wg % wg_per_slab;
  // Sample whose work-groups cover `rem`: last j with info[j].wg_prefix <= rem.
  int lo = 0, hi = n - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (info[mid].wg_prefix <= rem) lo = mid;
    else hi = mid - 1;
  }
  const MigrateInfo m = info[lo];
  const int64_t r2 = rem - m.wg_prefix;
  const int head = (int)(r2 / m.chunks), chunk = (int)(r2 % m.chunks);
  const int dc = head_dim / 8;
  const int64_t units = (int64_t)m.count * dc;       // 16-byte units of this run
  const int64_t u0 = (int64_t)chunk * kChunk;
  bf16* p = pool + m.kv_base + (((int64_t)lk * n_kv_heads + head) * m.cap + m.begin) * head_dim;
  bf16* b = buf + (((int64_t)lk * tok_total + m.tok_prefix) * n_kv_heads + (int64_t)head * m.count) *
                      head_dim;
  const i32x4* src = (const i32x4*)(TO_BUFFER ? p : b);
  i32x4* dst = (i32x4*)(TO_BUFFER ? b : p);
  i32x4 v[kPer];
#pragma unroll
  for (int k = 0; k < kPer; ++k) {
    const int64_t u = u0 + threadIdx.x + 256 * k;
    if (u < units) v[k] = src[u];
  }
#pragma unroll
  for (int k = 0; k < kPer; ++k) {
    const int64_t u = u0 + threadIdx.x + 256 * k;
    if (u < units) dst[u] = v[k];
  }
}

}  // namespace

int64_t kv_transfer_chunks(int count, int head_dim) {
  const int64_t units = (int64_t)count * (head_dim / 8);
  return units == 0 ? 0 : (units + kChunk - 1) / kChunk;
}

hipError_t launch_kv_transfer(bool to_buffer, const MigrateInfo* info, int n, int64_t wg_per_slab,
                              int tok_total, bf16* pool, bf16* buf, int n_layers, int n_kv_heads,
                              int head_dim, hipStream_t s) {
  if (wg_per_slab == 0) return hipSuccess;
  const int64_t grid = (int64_t)n_layers * 2 * wg_per_slab;
  if (grid > 0x7fffffff) return hipErrorInvalidValue;
  if (to_buffer)
    kv_transfer_kernel<true><<<(unsigned)grid, 256, 0, s>>>(info, n, wg_per_slab, tok_total, pool,
                                                            buf, n_kv_heads, head_dim);
  else
    kv_transfer_kernel<false><<<(unsigned)grid, 256, 0, s>>>(info, n, wg_per_slab, tok_total, pool,
                                                             buf, n_kv_heads, head_dim);
  return hipGetLastError();
}

}  // namespace spec
