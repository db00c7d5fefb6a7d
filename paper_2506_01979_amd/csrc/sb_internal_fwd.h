// Internal declarations of the forward path (host + device visible).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "sb_internal.h"

namespace sb {

enum { EPI_QKV = 0, EPI_RESID = 1, EPI_SWIGLU = 2, EPI_LOGITS = 3, EPI_RESID_NORM = 4 };

// Per-row tree metadata kept in the workspace.
struct Meta {
  int32_t pos[SB_MAX_ROWS];      // kv_len + depth(i)
  uint32_t anc[SB_MAX_ROWS][8];  // bit j: row j is on the path root..i
};

// Geometry of a packed weight kind.
struct PackGeom {
  int K;       // source columns
  int ks;      // packed k-steps (bf16: K padded to a multiple of 256)
  int tiles;   // 16-row tiles (bf16)
  int rows;    // output rows (natural-order kinds) / total rows (f32)
  size_t bytes;
};

inline int ceil_div(int a, int b) { return (a + b - 1) / b; }
inline int round_up(int a, int b) { return ceil_div(a, b) * b; }

inline PackGeom pack_geom(const sb_model_config &c, int kind) {
  PackGeom g{};
  const int H = c.hidden, d = c.head_dim, F = c.ffn;
  const int qd = c.n_heads * d, kvd = c.n_kv_heads * d;
  const bool bf = c.dtype == SB_BF16;
  switch (kind) {
    case SB_W_QKV:
      g.K = H;
      g.rows = qd + 2 * kvd;
      g.tiles = (qd + 2 * kvd) / 16;
      break;
    case SB_W_O:
      g.K = qd;
      g.rows = H;
      g.tiles = ceil_div(H, 16);
      break;
    case SB_W_GATE_UP:
      g.K = H;
      g.rows = 2 * F;
      g.tiles = round_up(F, 256) / 8;  // covers every column of the padded activation
      break;
    case SB_W_DOWN:
      g.K = F;
      g.rows = H;
      g.tiles = ceil_div(H, 16);
      break;
    case SB_W_LM_HEAD:
      g.K = H;
      g.rows = c.vocab;
      g.tiles = ceil_div(c.vocab, 16);
      break;
    default:
      return g;
  }
  if (bf) {
    g.ks = round_up(ceil_div(g.K, 32), 8);  // whole 8-k-step chunks
    g.bytes = (size_t)g.tiles * g.ks * 1024;
  } else {
    g.ks = g.K;
    g.bytes = (size_t)g.rows * g.K * sizeof(float);
  }
  return g;
}

struct EmbedArgs {
  const int32_t *tokens;
  const void *embed;
  float *h;
  int vocab, hidden, n_tok, kv_len;
  Meta *meta;
  float2 *rope;  // [n_tok][head_dim/2] cos, sin
  int head_dim;
  double theta[128];  // RoPE frequencies base^(-2j/d), j < head_dim/2
};

// Largest K split of a residual projection (slices of the delta buffer).
constexpr int kMaxSplit = 4;

struct GemmArgs {
  const uint16_t *W;   // packed weights
  const uint16_t *X;   // packed activations
  int ks;              // k-steps (a multiple of 8)
  int tiles;           // 16-row weight tiles
  int n_tok;           // valid activation rows
  int out_rows;        // RESID: hidden; LOGITS: vocab
  int epi;             // EPI_*
  int split, groups;   // K ranges, tile groups (grid = split * groups)
  float *h;            // RESID output: projection delta slices, fp32 [split][n_tok][out_rows]
  float *logits;       // LOGITS output
  uint16_t *act;       // SWIGLU output (packed, act_ks k-steps)
  int act_ks;
  uint16_t *q;         // QKV: q after RoPE, [rows][n_heads][head_dim]
  uint16_t *kc, *vc;   // QKV: this layer's cache [n_kv][cap][head_dim]
  int cap, kv_len;
  int n_heads, n_kv, head_dim;
  const float2 *rope;  // [rows][head_dim/2]
  // RESID_NORM (a residual projection fused with the following RMSNorm):
  // h, fp32 [n_tok][out_rows], is the residual stream itself and is updated
  // in place; the norm's input scaled by its gain, bf16(h * gain), is packed
  // into xn (xn_ks k-steps); ss[t][group] (kSsGroups per row) receives the
  // group's sum of h^2 over its rows for token t.
  const float *gain;
  uint16_t *xn;
  int xn_ks;
  float *ss;
  // Consumer of a RESID_NORM launch (X = its xn): every output of token t
  // is multiplied by 1 / sqrt(sum_{g < ss_groups} ss_in[t][g] / norm_dim + eps),
  // the RMSNorm scale applied after the projection.
  const float *ss_in;
  int ss_groups, norm_dim;
  float eps;
  // Otherwise, consumer of an RMSNorm kernel (X = bf16(h g)): every output
  // of token t is multiplied by rs_in[t] = 1/rms (QKV, SWIGLU, LOGITS).
  const float *rs_in;
  // LOGITS with the softmax statistics fused (lm_part not null): the
  // group's partial statistics of every token row, lm_part[t][groups], at
  // inverse temperature lm_inv_t (lm_greedy: T = 0).
  LmPart *lm_part;
  float lm_inv_t;
  int lm_greedy;
};

// Row stride of the per-(token, group) sums of squares of a RESID_NORM
// launch (its largest group count).
constexpr int kSsGroups = 256;
// Largest token count of a RESID_NORM launch and its consumer.
constexpr int kNormFuseRows = 128;

struct AttnArgs {
  const void *q;        // bf16 or f32 [rows][n_heads][d]
  const void *kc, *vc;  // this layer's cache [n_kv][cap][d]
  int cap, kv_len, n_tok, n_heads, n_kv, head_dim;
  int n_chunks;     // key ranges per KV head (attn_splits)
  const Meta *meta;
  float scale;
  float *part_o;   // [n_kv][n_chunks][R][d]
  float *part_ml;  // [n_kv][n_chunks][R][2]
};

// k_bf16.hip
hipError_t launch_pack_bf16(int kind, const sb_model_config &c, const void *src0, const void *src1,
                            const void *src2, void *dst, hipStream_t s);
hipError_t launch_embed_meta(const EmbedArgs &a, const TreeArg &tree, int blocks, int bf16,
                             hipStream_t s);
// Packs bf16(h g) and writes r = 1/rms per row to rs (nullable); tap
// (nullable, [n_tok][hidden] fp32) also receives the residual rows after
// the delta slices are added, or with tap_normed the normalised rows (h r) g.
hipError_t launch_rmsnorm_pack(float *h, const float *delta, int n_delta, const float *g,
                               int hidden, int ks, int n_tok, int n_pad, float eps, uint16_t *out,
                               float *rs, hipStream_t s, float *tap = nullptr,
                               int tap_normed = 0);
// H-RAD (k_hrad.hip): y1 = ReLU(W1 z + b1) into ws, then the 64-unit layer,
// the 3 logits and their argmax
struct HradArgs {
  const float *taps;  // [k][max_rows][hidden]
  int k, max_rows, hidden, vocab;
  const uint16_t *embed;  // bf16 [vocab][hidden]
  const sb_step_result *res;
  const float *w1, *b1, *w2, *b2, *w3, *b3;
  float *y1;  // [SB_HRAD_H1] workspace
  float *logits3;
  int32_t *cls;
};
hipError_t launch_hrad(const HradArgs &a, hipStream_t s);
// Branch-point candidates (k_branch.hip): the selection on one workgroup,
// then the carried rows
struct BranchArgs {
  const float *q;  // [vocab]
  const int32_t *x_b;
  int vocab, k_max, mode;
  int vec4;        // vocab % 4 == 0 and q, rows 16-byte aligned
  const float *u;  // [k_max]
  int32_t *count, *tokens;
  float *rows;     // [k_max][vocab]
  double *znorm;   // [SB_BRANCH_MAX_K] workspace: the mass before each draw
};
hipError_t launch_branch(const BranchArgs &a, hipStream_t s);
// Launch geometry of a GEMM: token tiles (rounded up to a kernel's), tiles per
// pass, K split, tile groups and grid.
// Largest tiles per pass of the GEMM kernel per token-tile count (its
// register budget), and the (tile, token tile) accumulator pairs it reduces
// per LDS round.
constexpr int gemm_nt_cap(int tt) {
  return tt <= 4 ? 8 : tt <= 6 ? 6 : tt <= 8 ? 4 : tt <= 12 ? 2 : 1;
}
constexpr int kRedPairs = 16;
struct GemmPlan {
  int tt, nt, split, groups, grid;
  int wide;  // k_gemm_wide with this many K parts per workgroup (0: k_gemm)
};
GemmPlan plan_gemm(int epi, int tiles, int ks, int n_tok);
// Launches of a planned GEMM, one per epilogue kind (k_gemm_*.hip).
hipError_t launch_gemm_qkv(const GemmArgs &a, const GemmPlan &p, hipStream_t s);
hipError_t launch_gemm_resid(const GemmArgs &a, const GemmPlan &p, hipStream_t s);
hipError_t launch_gemm_swiglu(const GemmArgs &a, const GemmPlan &p, hipStream_t s);
hipError_t launch_gemm_logits(const GemmArgs &a, const GemmPlan &p, hipStream_t s);
hipError_t launch_gemm_resid_norm(const GemmArgs &a, const GemmPlan &p, hipStream_t s);
// *split receives the K split used (the number of delta slices for RESID).
hipError_t launch_gemm(int epi, const GemmArgs &a, int tiles, int *split, hipStream_t s);
// Timing events a measured launch hands to the next GEMM dispatch, which
// passes them to hipExtLaunchKernelGGL so that the dispatch itself records
// the kernel's start and end; taken once, then ignored.
struct LaunchEvents {
  hipEvent_t start = nullptr, stop = nullptr;
  bool taken = true;
};
extern thread_local LaunchEvents g_launch_events;
// Whether a residual projection of `tiles` tiles over n_tok rows can run as
// RESID_NORM (one pass, one reduction round, at most kSsGroups groups,
// n_tok <= kNormFuseRows); *groups receives its group count.
bool resid_norm_fusable(int tiles, int ks, int n_tok, int *groups);

// k_attn.hip
// Key ranges per KV head: about kAttnTargetGroups workgroups in all, one per
// (KV head, key range, block of at most 16 kAttnMaxRowTiles query rows of
// the head's group).
constexpr int kAttnTargetGroups = 256;
constexpr int kAttnMinSteps = 4;
constexpr int kAttnMaxRowTiles = 3;  // 48-row blocks (64: 70B step 0.36 ms slower)
constexpr int kAttnCUs = 256;  // compute units the launch shape is planned for (MI355X)
int attn_row_tiles(int rows);
int attn_steps_per_wave(int n_kv, int head_dim, int nkeys, int rows);
bool attn_rb_split(int n_kv, int head_dim, int nkeys, int rows);
int attn_splits(int n_kv, int head_dim, int nkeys, int rows);
hipError_t launch_attn_bf16(const AttnArgs &a, hipStream_t s);
hipError_t launch_attn_merge_bf16(const AttnArgs &a, uint16_t *out_packed, int out_ks,
                                  hipStream_t s);

// ---- persistent forward (k_persist.hip) ------------------------------------
// One cooperative launch runs every layer of a bf16 verify forward: one
// 512-thread workgroup per compute unit, the phases of a layer separated by
// device-wide barriers, each GEMM's first weight loads issued before the
// barrier that precedes it.

// Per-layer weight pointers, read by the kernel from a device table.
struct PkLayer {
  const uint16_t *qkv, *o, *gu, *dn;
  const float *g_attn, *g_mlp;
};
// A GEMM of the persistent forward: packed weights, k-steps, 16-row tiles,
// tiles per pass, K split, tile groups.
struct PkGemmPlan {
  int ks, tiles, nt, split, groups;
};
// Barrier counters (one per XCD group of workgroups, 128 bytes apart) and
// the status word (non-zero: a barrier timed out, the step is invalid).
struct PkSync {
  unsigned grp[8][32];
  unsigned status[32];
};
struct PkArgs {
  int n_layers, hidden, n_heads, n_kv, head_dim, ffn, vocab;
  int n_tok, kv_len, cap;
  float eps, scale;
  PkGemmPlan qkv, o, gu, dn, lm;
  int n_chunks;              // attention key ranges per KV head
  int xa_ks, xo_ks, act_ks;  // k-steps of the packed activations
  const PkLayer *layers;     // [n_layers] device table
  const uint16_t *lm_head;
  const float *g_final;
  uint16_t *kc, *vc;         // layer 0 of the caches
  size_t layer_kv;           // elements per layer of one cache
  float *h, *delta, *ss, *part_o, *part_ml, *logits;
  uint16_t *xa, *xo, *act, *q;
  const Meta *meta;
  const float2 *rope;
  PkSync *sync;
};
// Layers whose table one k_pk_table launch writes (kernel arguments hold
// their pointers).
constexpr int kPkTableLayers = 64;
struct PkTableArgs {
  PkLayer layer[kPkTableLayers];
  PkLayer *dst;
  int n;
  PkSync *sync;  // zeroed by the first launch (nullptr for the others)
};
// Threads of a persistent workgroup; 32-key steps of an attention item.
constexpr int kPkThreadsHost = 512;
constexpr int kPkAttnMaxSteps = 16;
// Key ranges per KV head of the persistent attention phase (about one work
// item per workgroup, at most kPkAttnMaxSteps steps of 32 keys each).
int pk_attn_chunks(int n_kv, int nkeys, int nwg);
// Whether the persistent kernel runs this step, with its GEMM plans and
// kernel (nwg: workgroups = compute units).
bool pk_plan(const sb_model_config &c, int n_tok, int nwg, PkArgs *a, const void **kernel);
// Kernel of a signature: tt token tiles, rt query tiles per attention
// block, special = the 7B-shaped tiles per pass (null: not built).
const void *pk_kernel(int tt, int rt, bool special);
hipError_t launch_pk_table(const PkTableArgs &t, hipStream_t s);
hipError_t launch_persist(const PkArgs &a, const void *kernel, int grid, hipStream_t s);

// k_f32.hip
hipError_t launch_f32_rmsnorm(const float *h, const float *g, int hidden, int n_tok, float eps,
                              float *out, hipStream_t s);
hipError_t launch_f32_gemm(const float *X, const float *W, float *Y, int n_tok, int M, int K,
                           int ldy, int accumulate, hipStream_t s);
hipError_t launch_f32_rope_qkv(const float *qkv, const sb_model_config &c, int n_tok,
                               const float2 *rope, float *q, float *kc, float *vc, int cap,
                               int kv_len, hipStream_t s);
hipError_t launch_f32_attn(const AttnArgs &a, float *out, hipStream_t s);
hipError_t launch_f32_swiglu(const float *gu, int n_tok, int ffn, float *act, hipStream_t s);

}  // namespace sb
