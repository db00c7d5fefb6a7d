// KV rollback / compaction after the accept/resample walk.
//
// The paper keeps the branch whose branch point is accepted and discards the
// other branches together with their KV cache (Section "Branch Resampling",
// "Branch Verification").  The verify forward wrote tree row i to slot
// kv_len + i; here the rows on the accepted path move to the contiguous
// slots kv_len + j.  K is cached as [head][slot][d], V transposed as
// [head][d][slot]; the work walks j in ascending batches, and every batch
// reads its sources before it writes its destinations.  The source path[j]
// is >= j, so no slot is read after an earlier batch overwrote it; a K
// column or a V row is owned by one thread or by one 8-lane group of one
// wave, so no other work touches it.
#include "sb_device.h"
#include "sb_internal.h"

namespace sb {
namespace {

__device__ __forceinline__ int clamp_path(const sb_step_result *res, int kv_len, int capacity) {
  // a result that does not describe a path inside the cache moves nothing
  int plen = res->path_len;
  if (plen < 1 || plen > SB_MAX_ROWS || kv_len + plen > capacity) plen = 1;
  return plen;
}

// Path positions moved per batch.  K: a thread owns one 16-byte column of
// one (layer, KV head) and loads the sources of a whole batch (branch-free
// buffer loads; positions that move nothing read past the end) before it
// stores any.  V (transposed, 2-byte elements along the slot axis): the 8
// lanes of a group own one (layer, head, d) row, lane l the positions
// j0 + l, so a wave instruction touches 8 short runs of consecutive slots.
constexpr int kMoveBatch = 8;

template <typename T>
__global__ __launch_bounds__(256) void k_rollback(int k_cols, int vec_per_row, int v_rows,
                                                  int capacity, uint4 *__restrict__ k,
                                                  T *__restrict__ vt, int kv_len,
                                                  const sb_step_result *__restrict__ res,
                                                  int32_t *__restrict__ new_len) {
  // the path once into LDS: source row of every path position, -1 where
  // nothing moves (already in place, or outside the cache)
  __shared__ int s_src[SB_MAX_ROWS];
  __shared__ int s_plen;
  if (threadIdx.x == 0) s_plen = clamp_path(res, kv_len, capacity);
  __syncthreads();
  const int plen = s_plen;
  for (int j = threadIdx.x; j < plen; j += blockDim.x) {
    const int src = res->path[j];
    s_src[j] = (src <= j || kv_len + src >= capacity) ? -1 : src;
  }
  __syncthreads();
  if (blockIdx.x == 0 && threadIdx.x == 0) *new_len = kv_len + plen;
  const int total = k_cols + v_rows * kMoveBatch;
  const int vbytes = capacity * (int)sizeof(T);
  for (int c = blockIdx.x * blockDim.x + threadIdx.x; c < total; c += gridDim.x * blockDim.x) {
    if (c < k_cols) {
      const int head = c / vec_per_row;  // flattened (layer, kv head)
      const int col = c - head * vec_per_row;
      uint4 *base = k + (size_t)head * capacity * vec_per_row + col;
      const int kbytes = capacity * vec_per_row * 16;
      const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
          (void *)(k + (size_t)head * capacity * vec_per_row), 0, kbytes, kBufferDword3);
      for (int j0 = 1; j0 < plen; j0 += kMoveBatch) {
        i32x4 val[kMoveBatch];
#pragma unroll
        for (int b = 0; b < kMoveBatch; ++b) {
          const int j = j0 + b;
          const int src = j < plen ? s_src[j] : -1;
          const int off = src >= 0 ? ((kv_len + src) * vec_per_row + col) * 16 : kbytes;
          val[b] = __builtin_amdgcn_raw_buffer_load_b128(rs, off, 0, 0);
        }
#pragma unroll
        for (int b = 0; b < kMoveBatch; ++b) {
          const int j = j0 + b;
          if (j < plen && s_src[j] >= 0)
            base[(size_t)(kv_len + j) * vec_per_row] = __builtin_bit_cast(uint4, val[b]);
        }
      }
    } else {
      const int item = c - k_cols;
      T *row = vt + (size_t)(item / kMoveBatch) * capacity;  // one (layer, head, d) row
      const int lane8 = item % kMoveBatch;
      const __amdgpu_buffer_rsrc_t rs =
          __builtin_amdgcn_make_buffer_rsrc((void *)row, 0, vbytes, kBufferDword3);
      for (int j0 = 1; j0 < plen; j0 += kMoveBatch) {
        const int j = j0 + lane8;
        const int src = j < plen ? s_src[j] : -1;
        const int off = src >= 0 ? (kv_len + src) * (int)sizeof(T) : vbytes;
        if (sizeof(T) == 2) {
          const uint16_t x = (uint16_t)__builtin_amdgcn_raw_buffer_load_b16(rs, off, 0, 0);
          if (src >= 0) ((uint16_t *)row)[kv_len + j] = x;
        } else {
          const uint32_t x = __builtin_amdgcn_raw_buffer_load_b32(rs, off, 0, 0);
          if (src >= 0) ((uint32_t *)row)[kv_len + j] = x;
        }
      }
    }
  }
}

// The end of a SpecBranch round (Algorithm 2, verification phase): the
// target's walk over the trunk chain [root, x_1 .. x_c] and Algorithm 1 at
// the trunk's last row give the committed token; the draft cache keeps the
// root, the accepted trunk rows and, with a kept branch, that branch's rows
// whose KV the draft computed (depths 1 .. depth - 1).  One thread.
__global__ void k_round_finish(int chain, int branches, int depth, const sb_step_result *walk,
                               const int32_t *sel, sb_round_result *out, sb_step_result *dpath) {
  if (threadIdx.x != 0 || blockIdx.x != 0) return;
  const int n = walk->n_accepted;
  const bool whole = n >= chain;
  int kept = -1, token = walk->next_token, flags = walk->flags;
  if (whole && sel) {
    kept = sel[0] >= 0 && sel[0] < branches ? sel[0] : -1;
    token = sel[1];
    flags |= sel[2];
  }
  // the walk's bonus draw (a fully accepted trunk) is not a committed token
  // here: with candidates, Algorithm 1 decides; with none, the draw from
  // p at the trunk's last row is the token
  int len = 0;
  const int n_trunk = whole ? chain : n;
  for (int j = 0; j <= n_trunk; ++j) dpath->path[len++] = j;
  if (kept >= 0)
    for (int d = 1; d < depth; ++d) dpath->path[len++] = chain + 1 + (d - 1) * branches + kept;
  for (int j = len; j < SB_MAX_ROWS; ++j) dpath->path[j] = -1;
  dpath->n_accepted = len - 1;
  dpath->branch = kept;
  dpath->next_token = token;
  dpath->path_len = len;
  dpath->flags = flags;
  dpath->n_rejected = 0;
  dpath->bonus = 0;
  dpath->reserved = 0;
  out->n_trunk = n_trunk;
  out->kept = kept;
  out->token = token;
  out->flags = flags;
  out->draft_len = len;
  out->reserved[0] = out->reserved[1] = out->reserved[2] = 0;
}

}  // namespace

hipError_t launch_round_finish(int chain, int branches, int depth, const sb_step_result *walk,
                               const int32_t *sel, sb_round_result *out, sb_step_result *dpath,
                               hipStream_t s) {
  hipLaunchKernelGGL(k_round_finish, dim3(1), dim3(64), 0, s, chain, branches, depth, walk, sel,
                     out, dpath);
  return hipGetLastError();
}

hipError_t launch_rollback(int n_layers, int n_kv, int capacity, int head_dim, int elem_bytes,
                           void *k, void *v, int kv_len, const sb_step_result *res,
                           int32_t *new_len, hipStream_t s) {
  const int vec_per_row = head_dim * elem_bytes / 16;
  const int k_cols = n_layers * n_kv * vec_per_row;
  const int v_rows = n_layers * n_kv * head_dim;
  int blocks = (k_cols + v_rows * kMoveBatch + 255) / 256;
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
