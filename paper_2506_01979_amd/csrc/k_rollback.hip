// KV rollback / compaction after the accept/resample walk.
//
// The paper keeps the branch whose branch point is accepted and discards the
// other branches together with their KV cache (Section "Branch Resampling",
// "Branch Verification").  The verify forward wrote tree row i to slot
// kv_len + i; here the rows on the accepted path move to the contiguous
// slots kv_len + j.  Each thread owns one 16-byte column of one (layer, KV
// head) and walks j in ascending order: the source row path[j] is >= j, so
// no slot is read after an earlier step of the same thread overwrote it, and
// threads never share a column.
#include "sb_internal.h"

namespace sb {
namespace {

__global__ __launch_bounds__(256) void k_rollback(int n_cols, int vec_per_row, int capacity,
                                                  int row_vecs_stride, uint4 *__restrict__ k,
                                                  uint4 *__restrict__ v, int kv_len,
                                                  const sb_step_result *__restrict__ res,
                                                  int32_t *__restrict__ new_len) {
  // a result that does not describe a path inside the cache moves nothing
  int plen = res->path_len;
  if (plen < 1 || plen > SB_MAX_ROWS || kv_len + plen > capacity) plen = 1;
  if (blockIdx.x == 0 && threadIdx.x == 0) *new_len = kv_len + plen;
  for (int c = blockIdx.x * blockDim.x + threadIdx.x; c < n_cols; c += gridDim.x * blockDim.x) {
    const int head = c / vec_per_row;     // flattened (layer, kv head)
    const int col = c - head * vec_per_row;
    const size_t base = (size_t)head * capacity * row_vecs_stride + col;
    for (int j = 1; j < plen; ++j) {
      const int src = res->path[j];
      if (src == j || src < j || kv_len + src >= capacity) continue;
      const size_t s = base + (size_t)(kv_len + src) * row_vecs_stride;
      const size_t d = base + (size_t)(kv_len + j) * row_vecs_stride;
      k[d] = k[s];
      v[d] = v[s];
    }
  }
}

}  // namespace

hipError_t launch_rollback(int n_layers, int n_kv, int capacity, int row_bytes, void *k, void *v,
                           int kv_len, const sb_step_result *res, int32_t *new_len,
                           hipStream_t s) {
  const int vec_per_row = row_bytes / 16;
  const int n_cols = n_layers * n_kv * vec_per_row;
  int blocks = (n_cols + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(k_rollback, dim3(blocks), dim3(256), 0, s, n_cols, vec_per_row, capacity,
                     vec_per_row, (uint4 *)k, (uint4 *)v, kv_len, res, new_len);
  return hipGetLastError();
}

}  // namespace sb
