// KV rollback / compaction after the accept/resample walk.
//
// The paper keeps the branch whose branch point is accepted and discards the
// other branches together with their KV cache (Section "Branch Resampling",
// "Branch Verification").  The verify forward wrote tree row i to slot
// kv_len + i; here the rows on the accepted path move to the contiguous
// slots kv_len + j.  K is cached as [head][slot][d]: a thread owns one
// 16-byte column of one (layer, KV head).  V is cached transposed,
// [head][d][slot]: a thread owns one d-row.  Either way a thread walks j in
// ascending order; the source path[j] is >= j, so no slot is read after an
// earlier step of the same thread overwrote it, and threads never share
// data.
#include "sb_internal.h"

namespace sb {
namespace {

__device__ __forceinline__ int clamp_path(const sb_step_result *res, int kv_len, int capacity) {
  // a result that does not describe a path inside the cache moves nothing
  int plen = res->path_len;
  if (plen < 1 || plen > SB_MAX_ROWS || kv_len + plen > capacity) plen = 1;
  return plen;
}

template <typename T>
__global__ __launch_bounds__(256) void k_rollback(int k_cols, int vec_per_row, int v_rows,
                                                  int capacity, uint4 *__restrict__ k,
                                                  T *__restrict__ vt, int kv_len,
                                                  const sb_step_result *__restrict__ res,
                                                  int32_t *__restrict__ new_len) {
  const int plen = clamp_path(res, kv_len, capacity);
  if (blockIdx.x == 0 && threadIdx.x == 0) *new_len = kv_len + plen;
  const int total = k_cols + v_rows;
  for (int c = blockIdx.x * blockDim.x + threadIdx.x; c < total; c += gridDim.x * blockDim.x) {
    if (c < k_cols) {
      const int head = c / vec_per_row;  // flattened (layer, kv head)
      const int col = c - head * vec_per_row;
      const size_t base = (size_t)head * capacity * vec_per_row + col;
      for (int j = 1; j < plen; ++j) {
        const int src = res->path[j];
        if (src <= j || kv_len + src >= capacity) continue;
        k[base + (size_t)(kv_len + j) * vec_per_row] = k[base + (size_t)(kv_len + src) * vec_per_row];
      }
    } else {
      T *row = vt + (size_t)(c - k_cols) * capacity;  // one (layer, head, d) row
      for (int j = 1; j < plen; ++j) {
        const int src = res->path[j];
        if (src <= j || kv_len + src >= capacity) continue;
        row[kv_len + j] = row[kv_len + src];
      }
    }
  }
}

}  // namespace

hipError_t launch_rollback(int n_layers, int n_kv, int capacity, int head_dim, int elem_bytes,
                           void *k, void *v, int kv_len, const sb_step_result *res,
                           int32_t *new_len, hipStream_t s) {
  const int vec_per_row = head_dim * elem_bytes / 16;
  const int k_cols = n_layers * n_kv * vec_per_row;
  const int v_rows = n_layers * n_kv * head_dim;
  int blocks = (k_cols + v_rows + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  if (elem_bytes == 2)
    hipLaunchKernelGGL(k_rollback<uint16_t>, dim3(blocks), dim3(256), 0, s, k_cols, vec_per_row,
                       v_rows, capacity, (uint4 *)k, (uint16_t *)v, kv_len, res, new_len);
  else
    hipLaunchKernelGGL(k_rollback<float>, dim3(blocks), dim3(256), 0, s, k_cols, vec_per_row,
                       v_rows, capacity, (uint4 *)k, (float *)v, kv_len, res, new_len);
  return hipGetLastError();
}

}  // namespace sb
