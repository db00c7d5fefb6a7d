// Internal declarations shared by the HIP translation units of libsb.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "sb.h"

namespace sb {

// Tree passed by value to kernels (parents as int16, row 0 = root).
struct TreeArg {
  int32_t n;
  int16_t parent[SB_MAX_ROWS];
};

// ---- sampling (k_sampling.hip) --------------------------------------------
// invalid (nullable): a device word; non-zero marks every row non-finite
hipError_t launch_softmax_stats(int vocab, int n_rows, const float *logits, float temperature,
                                sb_row_stats *stats, hipStream_t s,
                                const unsigned *invalid = nullptr);
// Softmax statistics of logits rows whose columns are split over groups
// (the LM head's workgroups): for row t and group g, the largest logit of
// the group's columns, its lowest index (INT_MAX when none is above -inf)
// and, at T > 0, the float64 sum of fl32(exp(z_v - m)) over the group's
// columns with m = fl32(lmax / T) (0 when lmax is -inf).  A NaN or +inf
// logit makes sum NaN (at T = 0 too).
struct LmPart {
  float lmax;
  int32_t arg;
  double sum;
};
// One row per workgroup: the statistics of rows 0 .. n_rows - 1 from their
// groups' partials, part[row][groups] (at most 256 groups).
hipError_t launch_stats_finish(const LmPart *part, int groups, int n_rows, float temperature,
                               sb_row_stats *stats, hipStream_t s);
hipError_t launch_walk(int vocab, const TreeArg &tree, const int32_t *tokens, const float *logits,
                       const sb_row_stats *stats, float temperature, const float *q,
                       const float *u, sb_step_result *result, void *ws, hipStream_t s);
hipError_t launch_select(int vocab, const float *logits_row, const sb_row_stats *stats_row,
                         float temperature, int n_cand, const int32_t *cand_tokens,
                         const float *q, const float *u, int32_t *out, void *ws, hipStream_t s);
size_t sample_ws_bytes(int vocab);
// Rows of a draft sample call: logits/stats row src[i] -> token and q row dst[i].
struct DraftRows {
  int32_t n;
  int32_t src[SB_DRAFT_MAX_ROWS], dst[SB_DRAFT_MAX_ROWS];
};
size_t draft_ws_bytes(int vocab, int n);
hipError_t launch_draft_sample(int vocab, const DraftRows &rows, const float *logits,
                               const sb_row_stats *stats, float temperature, const float *u,
                               int32_t *tokens, float *q, void *ws, hipStream_t s,
                               float *conf = nullptr);
// A q row conditioned on confidence, in place (q / q(C) on C = {q >= eps}).
hipError_t launch_confident_row(float *q, int vocab, float eps, hipStream_t s);

// ---- rollback (k_rollback.hip) ---------------------------------------------
hipError_t launch_round_finish(int chain, int branches, int depth, const sb_step_result *walk,
                               const int32_t *sel, sb_round_result *out, sb_step_result *dpath,
                               hipStream_t s);
hipError_t launch_rollback(int n_layers, int n_kv, int capacity, int head_dim, int elem_bytes,
                           void *k, void *v, int kv_len, const sb_step_result *res,
                           int32_t *new_len, hipStream_t s);

}  // namespace sb
