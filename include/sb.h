/*
 * sb.h -- C ABI of the MI355X branch-verification step of SpecBranch
 * (arXiv 2506.01979).
 *
 * One verify step of the paper's target model: a forward of a Llama-style
 * decoder over a token tree whose rows share one prefix KV cache (the
 * verification phase of Algorithm 2 scores every draft position with one
 * target forward; Section "Branch Resampling" keeps the surviving branch and
 * drops the others with their KV), row softmax statistics, the lossless
 * accept/resample walk (Preliminaries, "Speculative Decoding"; Appendix,
 * Algorithm 1 "Branch Speculative Sampling") and KV rollback.  Around it:
 * H-RAD's feature tap and length predictor (Section "H-RAD") and the draft
 * side of a round -- branch-point candidates, the draft's q rows and
 * draws, and a whole drafting round on the draft model (Section "Branch
 * Resampling"; Algorithm 2's drafting).
 *
 * Conventions shared by every entry point:
 *  - "d_" pointers are device pointers, "h_" pointers host pointers.  The
 *    caller owns every buffer (weights, KV cache, logits, q, uniforms,
 *    workspace, results); the library keeps only the pointers it is given
 *    and, in sb_model_create, a small host-side model record.
 *  - Every call is asynchronous on the given HIP stream and allocates no
 *    device memory.  The drafting calls alone block the host
 *    (sb_draft_round, sb_draft_chain, sb_draft_branches, sb_spec_round): they
 *    read back the few values that shape the draft tree -- each chain
 *    draft's probability against the confidence threshold, and B -- since
 *    the next launches' shapes depend on them.  A model handle must not be
 *    used from two streams at once, and two calls that share a workspace
 *    must not overlap.
 *  - Errors a host can detect (null pointers, bad sizes, a malformed tree,
 *    too little KV capacity or workspace, unsupported shapes) return an
 *    SB_ERR_* code before anything is enqueued.  SB_ERR_HIP reports a failed
 *    launch.  Numeric conditions met on the device are reported in flag
 *    words (SB_FLAG_*), never as a trap.
 *  - The tree: row 0 is the root (the last committed token, whose KV is not
 *    yet cached); every other row is a draft token whose parent is an
 *    earlier row: h_parents[0] == -1 and 0 <= h_parents[i] < i.  Row i sits
 *    at position kv_len + depth(i) and its K/V go to cache slot
 *    kv_len + i.  At most SB_MAX_ROWS rows.
 */
#ifndef SB_H
#define SB_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SB_MAX_ROWS 256

typedef enum {
  SB_OK = 0,
  SB_ERR_INVALID_ARG = 1,   /* null pointer, non-positive size, bad enum */
  SB_ERR_TREE = 2,          /* parents not a rooted tree in row order */
  SB_ERR_CAPACITY = 3,      /* KV capacity or workspace too small */
  SB_ERR_DTYPE = 4,         /* dtype not supported for this call */
  SB_ERR_HIP = 5,           /* a HIP call or kernel launch failed */
  SB_ERR_UNSUPPORTED = 6    /* shape outside what the kernels handle */
} sb_status;

typedef enum { SB_F32 = 0, SB_BF16 = 1 } sb_dtype;

/* Decoder shape (the paper's Table 7 lists the Llama widths).  SB_BF16
 * models store weights and KV in bfloat16 and accumulate in float32;
 * SB_F32 models are float32 throughout.  rope_theta is the RoPE base,
 * rms_eps the RMSNorm epsilon. */
typedef struct {
  int32_t n_layers, hidden, n_heads, n_kv_heads, head_dim, ffn, vocab;
  float rope_theta, rms_eps;
  int32_t dtype; /* sb_dtype */
} sb_model_config;

/* Weight kinds for sb_pack_weight.  Sources are row-major [out][in]
 * matrices in the model dtype, as a Llama checkpoint stores them. */
typedef enum {
  SB_W_QKV = 0,     /* src0 = Wq [n_heads*head_dim][hidden], src1 = Wk, src2 = Wv
                       ([n_kv_heads*head_dim][hidden]) */
  SB_W_O = 1,       /* src0 = Wo [hidden][n_heads*head_dim] */
  SB_W_GATE_UP = 2, /* src0 = Wgate [ffn][hidden], src1 = Wup [ffn][hidden] */
  SB_W_DOWN = 3,    /* src0 = Wdown [hidden][ffn] */
  SB_W_LM_HEAD = 4  /* src0 = W_lm [vocab][hidden] (untied from the embedding) */
} sb_weight_kind;

/* Per-layer device pointers.  Norm gains are float32 [hidden]; the four
 * matrices are in the layout sb_pack_weight writes. */
typedef struct {
  const float *attn_norm;
  const void *qkv;
  const void *o;
  const float *mlp_norm;
  const void *gate_up;
  const void *down;
} sb_layer_weights;

typedef struct {
  const void *embed;               /* [vocab][hidden], model dtype, row-major */
  const float *final_norm;         /* [hidden] */
  const void *lm_head;             /* packed SB_W_LM_HEAD */
  const sb_layer_weights *layers;  /* host array of n_layers entries */
} sb_model_weights;

/* KV cache in the model dtype: k is [n_layers][n_kv_heads][capacity][head_dim]
 * (one key per row) and v is stored transposed, [n_layers][n_kv_heads]
 * [head_dim][capacity] (one value dimension per row), so attention reads both
 * with unit-stride vector loads along its own contraction.  capacity must be
 * a multiple of 8; slots [0, kv_len) hold the committed prefix. */
typedef struct {
  void *k;
  void *v;
  int32_t capacity;
} sb_kv_cache;

/* Softmax statistics of one logits row at temperature T (16 bytes):
 *   T > 0: zmax = max_v fl32(l_v * fl32(1/T)),
 *          total = sum_v fl32(exp(fl32(z_v - zmax))) in float64;
 *   T = 0: zmax = max_v l_v, total = 1.
 * argmax is the lowest index of the largest logit.  The target
 * distribution is p(v) = fl32(exp(z_v - zmax)) / total (T > 0) or the one-hot
 * at argmax (T = 0).  sb_verify_forward on a bf16 model takes the same terms
 * relative to the largest scaled logit of each 16-column block and rescales
 * them to zmax in float64 (its statistics are computed in the LM head's
 * epilogue): total then agrees with the sum above to about 1e-7 relative;
 * zmax and argmax are identical. */
typedef struct {
  float zmax;
  int32_t argmax;
  double total;
} sb_row_stats;

#define SB_FLAG_NONFINITE 1     /* a logits row holds NaN or Inf */
#define SB_FLAG_QZERO 2         /* a tested draft token had q(x) == 0 */
#define SB_FLAG_ZERO_RESIDUAL 4 /* a residual had no mass; p~ kept */

/* Result of one accept/resample walk (device-resident, written by
 * sb_accept_resample, read by sb_kv_rollback). */
typedef struct {
  int32_t n_accepted;  /* accepted draft rows on the kept path */
  int32_t branch;      /* ordinal of the kept child of the root, -1 if none */
  int32_t next_token;  /* residual draw, or bonus draw after a full accept */
  int32_t path_len;    /* 1 + n_accepted */
  int32_t flags;       /* SB_FLAG_* */
  int32_t n_rejected;  /* candidate tests that failed along the walk */
  int32_t bonus;       /* 1 if next_token came from p of an accepted leaf */
  int32_t reserved;
  int32_t path[SB_MAX_ROWS]; /* rows root .. last accepted, by depth */
} sb_step_result;

/* Outcome of one SpecBranch round (sb_round_finish, device-resident). */
typedef struct {
  int32_t n_trunk;   /* accepted trunk drafts (0 .. chain) */
  int32_t kept;      /* kept branch (candidate index), or -1 */
  int32_t token;     /* the committed token after the accepted trunk: the
                        kept candidate, or a residual draw */
  int32_t flags;     /* SB_FLAG_* of the walk and the selection */
  int32_t draft_len; /* rows of the draft tree the draft cache keeps */
  int32_t reserved[3];
} sb_round_result;

typedef struct sb_model sb_model;

const char *sb_status_string(sb_status s);
int32_t sb_version(void);

/* ---- weights -------------------------------------------------------- */

/* Bytes of the packed form of one weight kind (0 for a bad config/kind). */
size_t sb_packed_bytes(const sb_model_config *cfg, int32_t kind);

/* Re-lays one weight kind into the kernels' layout: for SB_BF16, 16-row x
 * 32-column tiles in the operand order of the gfx950 bf16 matrix-core
 * instruction (rows padded to 16 and columns to a multiple of 256 -- whole
 * chunks of 8 k-steps -- with zeros; Q/K rows of
 * every head reordered so a tile holds RoPE pairs (j, j + d/2); gate and up
 * rows interleaved 8 by 8); for SB_F32, the source rows concatenated
 * (Wq;Wk;Wv and Wgate;Wup).  src* and dst are device pointers, dst holds
 * sb_packed_bytes(cfg, kind) bytes and must not alias a source. */
sb_status sb_pack_weight(const sb_model_config *cfg, int32_t kind, const void *src0,
                         const void *src1, const void *src2, void *dst, hipStream_t stream);

/* Records the config and the device weight pointers (not copied; they must
 * outlive the model).  No device memory is allocated. */
sb_status sb_model_create(const sb_model_config *cfg, const sb_model_weights *w,
                          sb_model **out);
void sb_model_destroy(sb_model *m);

/* ---- the verify step ------------------------------------------------ */

/* Workspace bytes sb_verify_forward needs for up to max_rows rows. */
size_t sb_workspace_bytes(const sb_model *m, int32_t max_rows, int32_t max_kv_len);

/* Target forward over the token tree (verification phase of Algorithm 2,
 * with every branch scored in one pass under a branch-causal mask).
 *   kv:        prefix cache; slots [0, kv_len) are read, tree row i's K/V
 *              are written to slot kv_len + i (needs kv_len + n_rows <=
 *              capacity).
 *   d_tokens:  [n_rows] token ids (row 0 = root).
 *   h_parents: [n_rows] host array, the tree (see top of file).
 *   temperature: T >= 0 for the statistics written to d_stats.
 *   d_logits:  [n_rows][vocab] float32 output.
 *   d_stats:   [n_rows] output (sb_row_stats at T).
 *   d_ws:      workspace of at least sb_workspace_bytes(m, n_rows, kv_len)
 *              bytes (ws_bytes). */
sb_status sb_verify_forward(sb_model *m, const sb_kv_cache *kv, int32_t kv_len,
                            const int32_t *d_tokens, const int32_t *h_parents, int32_t n_rows,
                            float temperature, float *d_logits, sb_row_stats *d_stats,
                            void *d_ws, size_t ws_bytes, hipStream_t stream);

/* ---- the verify forward without a workspace argument -------------------
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation).
 * Same computation, arguments and results as sb_verify_forward, with the
 * workspace taken from a file-scope device array of the library of
 * SB_NOALLOC_SCRATCH_BYTES bytes (128 MiB), one per device, allocated when
 * the library's code is loaded on that device and held until the process
 * ends.  The call allocates nothing: its first call on a device (with that
 * device current) looks the array's address up once.
 * Errors: SB_ERR_CAPACITY when the step needs more workspace than the
 * array holds (sb_workspace_bytes(m, n_rows, kv_len) >
 * SB_NOALLOC_SCRATCH_BYTES), before anything is enqueued; otherwise the
 * errors of sb_verify_forward.
 * Every call on one device shares that device's array: calls that overlap
 * on a device (two streams, two threads) race and must be serialised by
 * the caller.  The array keeps the last call's contents; every value the
 * forward reads from it is written earlier in the same call. */
#define SB_NOALLOC_SCRATCH_BYTES (128 * 1024 * 1024)
#define SB_NOALLOC_MAX_DEVICES 64
sb_status sb_verify_forward_noalloc(sb_model *m, const sb_kv_cache *kv, int32_t kv_len,
                                    const int32_t *d_tokens, const int32_t *h_parents,
                                    int32_t n_rows, float temperature, float *d_logits,
                                    sb_row_stats *d_stats, hipStream_t stream);

/* Row softmax statistics of [n_rows][vocab] float32 logits at T >= 0, as a
 * pass of its own over given logits (the verify step computes them in its
 * LM head's epilogue). */
sb_status sb_softmax_stats(int32_t vocab, int32_t n_rows, const float *d_logits,
                           float temperature, sb_row_stats *d_stats, hipStream_t stream);

/* Workspace bytes of sb_select_branch / sb_accept_resample for a vocab. */
size_t sb_sample_workspace_bytes(int32_t vocab);

/* Algorithm 1 (Branch Speculative Sampling) at one node.
 *   d_logits_row/d_stats_row: the node's target row and its statistics at T.
 *   d_cand_tokens: [n_cand] candidates in test order; d_q: [n_cand][vocab]
 *   float32, row i the distribution candidate i was drawn from (i.i.d.
 *   draws: the same row; top-k without replacement: the renormalised
 *   remainder; deterministic top-k: one-hot).  d_u: [n_cand + 1] uniforms
 *   in [0,1): u[i] tests candidate i, u[n_cand] drives the final draw.
 *   d_out: int32[3] = {accepted candidate index or -1, emitted token, flags}.
 * Accept iff float64(u) < p~(x) / float64(q(x)); after a rejection
 * p~ <- max(0, p~ - q_i) / Z (float64); with no acceptance the token is the
 * inverse-CDF draw min{v : C_v > u * C_last}. */
sb_status sb_select_branch(int32_t vocab, const float *d_logits_row,
                           const sb_row_stats *d_stats_row, float temperature, int32_t n_cand,
                           const int32_t *d_cand_tokens, const float *d_q, const float *d_u,
                           int32_t *d_out, void *d_ws, size_t ws_bytes, hipStream_t stream);

/* The accept/resample walk over the whole tree: from the root, Algorithm 1
 * over a node's children in ascending row order (the chain test where there
 * is one child); an accepted child becomes the node; when a leaf is reached
 * the bonus token is drawn from its p, otherwise from the residual.
 *   d_tokens: [n_rows]; h_parents: [n_rows] host tree;
 *   d_logits / d_stats: the verify forward's outputs at T;
 *   d_q: [n_rows][vocab] float32, row i the distribution draft row i was
 *   drawn from (row 0 unused);
 *   d_u: [n_rows] uniforms in [0,1): u[i] tests draft row i, u[0] drives the
 *   final draw;
 *   d_result: one sb_step_result (device). */
sb_status sb_accept_resample(int32_t vocab, int32_t n_rows, const int32_t *d_tokens,
                             const int32_t *h_parents, const float *d_logits,
                             const sb_row_stats *d_stats, float temperature, const float *d_q,
                             const float *d_u, sb_step_result *d_result, void *d_ws,
                             size_t ws_bytes, hipStream_t stream);

/* How sb_verify_forward runs a bf16 model (the results are the same to the
 * bf16 tolerance; float32 models always use the kernel chain):
 *   SB_FWD_AUTO        the chain of kernels (the faster form on MI355X);
 *   SB_FWD_KERNELS     a chain of kernels, several per layer;
 *   SB_FWD_PERSISTENT  the persistent forward: every layer and the LM head
 *                      in one cooperative launch of one workgroup per
 *                      compute unit, phases separated by device-wide
 *                      barriers; steps it does not fit return
 *                      SB_ERR_UNSUPPORTED.
 * A barrier of the persistent forward that does not complete within 2 s
 * ends the launch; the step's logits are then not valid and its row
 * statistics are NaN (SB_FLAG_NONFINITE in the walk).  New models start in
 * SB_FWD_AUTO.  The H-RAD tap is written by the chain only: while a tap is
 * set, SB_FWD_PERSISTENT runs the chain. */
#define SB_FWD_AUTO 0
#define SB_FWD_KERNELS 1
#define SB_FWD_PERSISTENT 2
sb_status sb_model_set_forward(sb_model *m, int32_t mode);

/* KV rollback (Section "Branch Resampling": non-selected branches and their
 * KV are discarded): copies the K/V of the rows on d_result->path from slot
 * kv_len + path[j] to slot kv_len + j for j = 0..path_len-1, in ascending j,
 * and writes kv_len + path_len to *d_new_len.  kv_len must be the value
 * given to the verify forward that wrote the tree rows. */
sb_status sb_kv_rollback(const sb_model *m, const sb_kv_cache *kv, int32_t kv_len,
                         const sb_step_result *d_result, int32_t *d_new_len,
                         hipStream_t stream);

/* ---- H-RAD: the draft-length predictor's features and MLP ------------ */

/* Hidden widths of H-RAD's MLP (Appendix, "H-RAD Training"). */
#define SB_HRAD_H1 256
#define SB_HRAD_H2 64
#define SB_HRAD_CLASSES 3

/* Feature tap of H-RAD (Section "H-RAD", z_t): while set, every
 * sb_verify_forward of this model also writes its last k_layers hidden
 * states, float32 d_taps[k][row][hidden] with k = 0 the layer
 * n_layers - k_layers (rows of the call's tree, at most max_rows of them;
 * a call with more rows returns SB_ERR_CAPACITY): for k < k_layers - 1 the
 * residual stream after that layer, for the last one the final RMSNorm's
 * output RMSNorm(h) * g_final (the last hidden state in the form a library
 * Llama model reports it).  d_taps = NULL clears the tap.  SB_BF16 models
 * only (SB_ERR_DTYPE otherwise); 1 <= k_layers <= n_layers.  While a tap is
 * set the forward runs as the chain of kernels (SB_FWD_KERNELS). */
sb_status sb_model_set_tap(sb_model *m, float *d_taps, int32_t k_layers, int32_t max_rows);

/* H-RAD's MLP weights, float32 device arrays, y = W x + b per layer:
 * w1 [SB_HRAD_H1][(k_layers + 1) * hidden], w2 [SB_HRAD_H2][SB_HRAD_H1],
 * w3 [SB_HRAD_CLASSES][SB_HRAD_H2]; biases of the output widths. */
typedef struct {
  const float *w1, *b1, *w2, *b2, *w3, *b3;
} sb_hrad_weights;

/* Workspace bytes of sb_hrad_predict. */
size_t sb_hrad_workspace_bytes(void);

/* H-RAD's class for the next round (Section "H-RAD", eqs. z_t, s_t):
 * z = Concat(the k_layers tapped hidden states of row r, the embedding of
 * token y), r = the last row of d_result->path (the last accepted
 * position) and y = d_result->next_token, through ReLU(W1 z + b1),
 * ReLU(W2 . + b2), W3 . + b3.  Writes the three logits to d_logits3 and
 * s_t = their argmax (lowest index on ties: 0 all reject, 1 use the
 * draft's confidence, 2 all accept) to *d_class.  d_taps as filled by the
 * forward that d_result's walk scored (k_layers, max_rows as given to
 * sb_model_set_tap); a path row >= max_rows or a token outside the
 * vocabulary yields class -1 and zero logits.  float32 arithmetic. */
sb_status sb_hrad_predict(const sb_model *m, const float *d_taps, int32_t k_layers,
                          int32_t max_rows, const sb_step_result *d_result,
                          const sb_hrad_weights *w, float *d_logits3, int32_t *d_class,
                          void *d_ws, size_t ws_bytes, hipStream_t stream);

/* ---- branch-point candidates (draft side) --------------------------- */

/* Candidate rules of sb_branch_candidates. */
typedef enum {
  SB_BRANCH_TOPK = 0, /* the B largest entries of q, one-hot rows */
  SB_BRANCH_IID = 1,  /* B independent inverse-CDF draws, each carrying q */
  SB_BRANCH_WOR = 2   /* draws without replacement, each carrying its remainder */
} sb_branch_mode;

#define SB_BRANCH_MAX_K 16
#define SB_BRANCH_MAX_VOCAB 1048576

/* Workspace bytes of sb_branch_candidates. */
size_t sb_branch_workspace_bytes(void);

/* Sibling first tokens at a branch point (Section "Branch Resampling"):
 * B = max(1, floor(k_max (1 - q[x_b]))) computed in float64 from the float32
 * q[x_b], at most the number of tokens with q > 0 (B = 0 when there are
 * none).  *d_x_b: the draft's token at the branch position, read on the
 * device (a value outside the vocabulary counts as q[x_b] = 0).
 * d_q: float32 [vocab], the draft's distribution at the branch
 * position (finite, non-negative; other values give unspecified candidates,
 * never a fault).  Each candidate carries the distribution it was drawn
 * from, which verification (Algorithm 1) subtracts from p:
 *  - SB_BRANCH_TOPK: the B largest entries, in descending order, lowest
 *    index first among equal values; row i is one-hot at token i;
 *  - SB_BRANCH_IID: token i is the first v whose float64 running sum of q
 *    over 0..v exceeds d_u[i] times the total; row i is q;
 *  - SB_BRANCH_WOR: the same draw over q with candidates 0..i-1 zeroed;
 *    row i is that remainder r divided by its float64 mass, float32(r_v / Z).
 * d_u: float32 [k_max] uniforms in [0, 1) (unused, may be NULL, for TOPK).
 * Outputs: *d_count = B; d_tokens[k_max] (entries B.. set to -1);
 * d_rows float32 [k_max][vocab], rows 0..B-1 written, the rest untouched.
 * Draws sum in a tree order, so a u within rounding of a boundary of the
 * running sum may pick the neighbouring token.  1 <= k_max <= SB_BRANCH_MAX_K,
 * 1 <= vocab <= SB_BRANCH_MAX_VOCAB, else SB_ERR_INVALID_ARG;
 * ws_bytes below sb_branch_workspace_bytes() gives SB_ERR_CAPACITY.  No
 * model is involved. */
sb_status sb_branch_candidates(const float *d_q, int32_t vocab, const int32_t *d_x_b, int32_t k_max,
                               int32_t mode, const float *d_u, int32_t *d_count,
                               int32_t *d_tokens, float *d_rows, void *d_ws, size_t ws_bytes,
                               hipStream_t stream);

/* ---- the draft side of a round ----------------------------------------- */

#define SB_DRAFT_MAX_ROWS 64

/* The draft's rows: for i < n, the distribution of logits row h_src_rows[i]
 * at T -- the p(v) the verify step defines, stored as float32 because that
 * row is what verification reads as q -- is written to row h_dst_rows[i] of
 * d_q, and the token drawn from those float32 values with d_u[i] (the first
 * v whose float64 running sum in vocabulary order exceeds d_u[i] times their
 * total) to d_tokens[h_dst_rows[i]].  T = 0: q is one-hot at the row's
 * argmax, which is the token.  d_logits: float32 [n_logit_rows][vocab] with
 * d_stats their sb_row_stats at the same T (as sb_verify_forward and
 * sb_softmax_stats write them; finite logits); d_tokens: int32
 * [n_out_rows]; d_q: float32 [n_out_rows][vocab]; d_ws of at least
 * sb_draft_sample_workspace_bytes(vocab, n) bytes (SB_ERR_CAPACITY).
 * 1 <= n <= SB_DRAFT_MAX_ROWS, 0 <= h_src_rows[i] < n_logit_rows,
 * 0 <= h_dst_rows[i] < n_out_rows and distinct, T >= 0, else
 * SB_ERR_INVALID_ARG.  The draw sums in blocks of 2048 tokens, so a u within
 * rounding of a boundary of the running sum may pick the neighbouring token. */
sb_status sb_draft_sample(int32_t vocab, int32_t n, const float *d_logits,
                          const sb_row_stats *d_stats, int32_t n_logit_rows,
                          const int32_t *h_src_rows, float temperature, const float *d_u,
                          int32_t *d_tokens, float *d_q, int32_t n_out_rows,
                          const int32_t *h_dst_rows, void *d_ws, size_t ws_bytes,
                          hipStream_t stream);

/* Workspace bytes of sb_draft_sample (per-block sums of each row). */
size_t sb_draft_sample_workspace_bytes(int32_t vocab, int32_t n);

/* Workspace bytes of sb_draft_round (0 for arguments it rejects). */
size_t sb_draft_round_workspace_bytes(const sb_model *draft, int32_t k_max, int32_t depth,
                                      int32_t trunk_max, int32_t kv_len);

/* One drafting phase of a SpecBranch round (Section "Branch Resampling";
 * the drafting of Algorithm 2, which marks a drafted token whose own
 * probability is below a threshold) on the draft model's prefix cache
 * (kv_len slots):
 *  1. the draft scores the root (d_tokens[0] on entry: the last committed
 *     token, whose KV is not yet cached) and drafts a chain: x_t (t = 1,
 *     2, ...) is drawn from the distribution at row t - 1 with d_u[t - 1].
 *     The branch point x_b is the first x_t with q(x_t) < confidence (both
 *     float32), or x_trunk_max; the c = t - 1 confident drafts before it
 *     stay as a chain in rows 1 .. c.  trunk_max = 1: x_b = x_1, c = 0;
 *  2. sb_branch_candidates spawns B first tokens by `mode` from the
 *     distribution x_b was drawn from, with d_u[trunk_max .. trunk_max +
 *     k_max - 1]; they replace x_b;
 *  3. each branch continues on its own path: its depth-d token (d = 2 ..
 *     depth) is drawn by sb_draft_sample from the draft's distribution at
 *     its depth d - 1 row, with d_u[trunk_max + k_max (d - 1) + i] for
 *     branch i; every step is one sb_verify_forward of the draft over the
 *     tree so far.
 * Rows: 0 the root, 1 .. c the chain (parent t - 1), then the branches
 * depth-major: row c + 1 + (d - 1) B + i is branch i's depth-d token, its
 * parent row c at d = 1 and row - B after that.  Outputs: d_tokens[1 .. c +
 * B depth] (int32 [trunk_max + k_max depth]; later entries may be
 * overwritten), d_q float32 [trunk_max + k_max depth][vocab] (row i the
 * distribution token i was drawn from; row 0 the branch position's, that of
 * x_b), h_parents[0 .. c + B depth] (host, [trunk_max + k_max depth]),
 * *h_branches = B, *h_chain = c.  The draft's cache slots kv_len .. are
 * written (capacity at least kv_len + trunk_max + k_max depth).  d_u:
 * float32 [trunk_max + k_max depth].  Blocks the host once per chain draft
 * before the last allowed one (to read its probability; not when confidence
 * <= 0, which every draft meets) and once to read B.
 * 1 <= k_max <= SB_BRANCH_MAX_K, depth >= 1, trunk_max >= 1, trunk_max +
 * k_max depth <= SB_MAX_ROWS, confidence not NaN. */
sb_status sb_draft_round(sb_model *draft, const sb_kv_cache *kv, int32_t kv_len, int32_t k_max,
                         int32_t mode, int32_t depth, int32_t trunk_max, float confidence,
                         float temperature, const float *d_u, int32_t *d_tokens, float *d_q,
                         int32_t *h_parents, int32_t *h_branches, int32_t *h_chain, void *d_ws,
                         size_t ws_bytes, hipStream_t stream);

/* The two phases of sb_draft_round as separate calls, so that the target
 * can verify the chain while the draft spawns the branches (Algorithm 2:
 * the DRAFTING phase drafts the chain; in the VERIFICATION phase the draft
 * branches at x_b while the target verifies the chain).
 * sb_draft_chain: step 1 of sb_draft_round -- d_tokens[0] the root on entry;
 *   rows 1 .. c of d_tokens / d_q the confident chain, row 0 of d_q the
 *   distribution x_b was drawn from, *d_xb (device int32) = x_b,
 *   *h_chain = c; d_u float32 [trunk_max]; d_tokens and d_q have at least
 *   trunk_max + 1 rows; d_ws of sb_draft_round_workspace_bytes(draft, 1, 1,
 *   trunk_max, kv_len) bytes.  Blocks the host once per chain draft before
 *   the last allowed one when confidence > 0.
 * sb_draft_branches: steps 2 and 3 of sb_draft_round after a chain of
 *   `chain` rows (rows 0 .. chain of d_tokens, row 0 of d_q as
 *   sb_draft_chain leaves them, d_xb): the candidates into rows chain + 1
 *   .. chain + B, the continuations depth-major after them; d_u float32
 *   [k_max depth] (candidates first, then one per branch per depth, as
 *   d_u + trunk_max of sb_draft_round); h_parents[0 .. chain + B depth],
 *   *h_branches = B; d_ws of sb_draft_round_workspace_bytes(draft, k_max,
 *   depth, chain + 1, kv_len) bytes.  Blocks the host once, to read B.
 * The draft's cache slots kv_len .. are written by both, as sb_draft_round
 * writes them.  Errors as sb_draft_round.
 * flags of sb_draft_chain: 0, or SB_CHAIN_CONDITIONED: each confident chain
 *   draft's q row is replaced by q conditioned on confidence, q(v) / q(C) on
 *   C = {v : q(v) >= confidence} and 0 elsewhere (q(C) the float64 sum of
 *   C's float32 values, each quotient rounded once to float32).  A draft is
 *   kept in the chain only when its own probability reaches the threshold,
 *   so it was in effect drawn from that row; testing it against the row
 *   keeps the round exactly lossless at any threshold, where Algorithm 2's
 *   test against the unconditioned q row does not when the chain's length
 *   depends on the drafts.  Other bits: SB_ERR_INVALID_ARG. */
#define SB_CHAIN_CONDITIONED 1
sb_status sb_draft_chain(sb_model *draft, const sb_kv_cache *kv, int32_t kv_len, int32_t trunk_max,
                         float confidence, int32_t flags, float temperature, const float *d_u,
                         int32_t *d_tokens, float *d_q, int32_t *d_xb, int32_t *h_chain,
                         void *d_ws, size_t ws_bytes, hipStream_t stream);
sb_status sb_draft_branches(sb_model *draft, const sb_kv_cache *kv, int32_t kv_len, int32_t chain,
                            const int32_t *d_xb, int32_t k_max, int32_t mode, int32_t depth,
                            float temperature, const float *d_u, int32_t *d_tokens, float *d_q,
                            int32_t *h_parents, int32_t *h_branches, void *d_ws, size_t ws_bytes,
                            hipStream_t stream);

/* The end of one SpecBranch round (Algorithm 2, verification phase;
 * Section "Branch Resampling", "Branch Verification").  The round verified
 * the chain [root, x_1 .. x_chain] with the target (d_walk: its
 * sb_accept_resample result over that chain) and, when the whole chain is
 * accepted, tests the `branches` candidates with Algorithm 1 at the chain's
 * last row (d_select: sb_select_branch's {candidate or -1, token, flags};
 * may be NULL when branches = 0).  Writes d_round: n_trunk = accepted
 * chain drafts; with a rejection inside the chain, token = the walk's
 * residual draw and kept = -1 (the branches are discarded); with the whole
 * chain accepted, no bonus token is drawn: kept / token are Algorithm 1's
 * (with no candidates, the token is the walk's draw from p at the last
 * row).  d_draft_path: an sb_step_result whose path is the draft tree's
 * kept rows -- the root, the accepted chain rows and, with a kept branch,
 * that branch's rows at depths 1 .. depth - 1 (the ones the draft's cache
 * holds KV for) -- for sb_kv_rollback of the draft's cache.  The target's
 * cache is rolled back with d_walk itself.  0 <= chain, 0 <= branches,
 * depth >= 1, 1 + chain + branches depth <= SB_MAX_ROWS. */
sb_status sb_round_finish(int32_t chain, int32_t branches, int32_t depth,
                          const sb_step_result *d_walk, const int32_t *d_select,
                          sb_round_result *d_round, sb_step_result *d_draft_path,
                          hipStream_t stream);

/* ---- one whole SpecBranch round on two streams ------------------------ */

/* Parameters of a round: the drafting phase's (sb_draft_round's k_max,
 * mode, depth, trunk_max, confidence), the temperature T >= 0 of both
 * models' distributions, and flags for sb_draft_chain (0 or
 * SB_CHAIN_CONDITIONED). */
typedef struct {
  int32_t k_max, mode, depth, trunk_max;
  float confidence, temperature;
  int32_t flags;
} sb_round_params;

/* Workspace bytes of sb_spec_round (0 for arguments it rejects). */
size_t sb_spec_round_workspace_bytes(const sb_model *target, const sb_model *draft,
                                     const sb_round_params *p, int32_t t_len, int32_t d_len);

/* One round of Algorithm 2 (a drafting phase, then the verification phase
 * that consumes it; Section "Branch Resampling", "Branch Verification"):
 *  1. on draft_stream, sb_draft_chain: the draft scores the root
 *     (d_tokens[0] on entry, the last committed token, cached by neither
 *     model) on its cache (d_len slots) and drafts the confident chain
 *     x_1 .. x_c and the branch point x_b;
 *  2. on verify_stream, once the chain is drafted: the target's
 *     sb_verify_forward over [root, x_1 .. x_c] (rows 0 .. c of d_logits /
 *     d_stats) and sb_accept_resample over that chain (d_walk; uniforms
 *     d_u_walk[0 .. c]); meanwhile, on draft_stream, sb_draft_branches
 *     spawns the candidates at x_b and extends them (d_u_draft +
 *     trunk_max);
 *  3. on verify_stream, once both are done: sb_select_branch at row c over
 *     the candidates (d_select; uniforms d_u_sel[0 .. B]), sb_round_finish
 *     (d_round), and the rollbacks of the target's cache (with d_walk) and
 *     of the draft's cache (the rows sb_round_finish keeps); d_new_lens =
 *     {target's new length, draft's new length}.
 * Buffers: d_u_draft float32 [trunk_max + k_max depth]; d_u_walk float32
 * [trunk_max + 1]; d_u_sel float32 [k_max + 1]; d_tokens int32 and d_q
 * float32 [trunk_max + k_max depth]([vocab]) as sb_draft_round fills them;
 * d_logits float32 [trunk_max][vocab]; d_stats [trunk_max]; d_walk one
 * sb_step_result; d_select int32 [3] (written when B > 0); d_round one
 * sb_round_result; d_new_lens int32 [2]; h_parents host int32
 * [trunk_max + k_max depth] (the draft tree, 1 + c + B depth entries);
 * *h_chain = c, *h_branches = B; d_ws of sb_spec_round_workspace_bytes.
 * Needs t_len + trunk_max <= the target cache's capacity and d_len +
 * trunk_max + k_max depth <= the draft cache's; both models share the
 * vocabulary and are distinct objects.  The two streams may be the same
 * stream (a serial round, same results bit for bit).  Blocks the host as
 * sb_draft_chain and sb_draft_branches do.  On return every part of the
 * round is ordered before verify_stream's later work; draft_stream holds
 * none of it.  Errors as the calls it makes. */
sb_status sb_spec_round(sb_model *target, const sb_kv_cache *t_kv, int32_t t_len, sb_model *draft,
                        const sb_kv_cache *d_kv, int32_t d_len, const sb_round_params *p,
                        const float *d_u_draft, const float *d_u_walk, const float *d_u_sel,
                        int32_t *d_tokens, float *d_q, float *d_logits, sb_row_stats *d_stats,
                        sb_step_result *d_walk, int32_t *d_select, sb_round_result *d_round,
                        int32_t *d_new_lens, int32_t *h_parents, int32_t *h_chain,
                        int32_t *h_branches, void *d_ws, size_t ws_bytes,
                        hipStream_t verify_stream, hipStream_t draft_stream);


/* ---- measurement ---------------------------------------------------- */

/* Kernel classes of the verify step, for sb_timer_start. */
typedef enum {
  SB_KC_QKV = 0,        /* QKV GEMM + RoPE + KV write */
  SB_KC_O = 1,          /* O GEMM + residual */
  SB_KC_GATE_UP = 2,    /* gate/up GEMM + SwiGLU */
  SB_KC_DOWN = 3,       /* down GEMM + residual */
  SB_KC_LM_HEAD = 4,    /* LM head GEMM */
  SB_KC_ATTN = 5,       /* branch-masked attention */
  SB_KC_ATTN_MERGE = 6, /* attention chunk merge */
  SB_KC_NORM = 7,       /* RMSNorm */
  SB_KC_STATS = 8,      /* softmax statistics */
  SB_KC_PERSIST = 9     /* the persistent forward (every layer + LM head) */
} sb_kernel_class;

/* Starts timing one kernel class of this model: every later launch of that
 * class by sb_verify_forward is bracketed by a pair of HIP events recorded on
 * the call's stream (at most `capacity` launches).  The events are created
 * here (host runtime objects, no device memory). */
sb_status sb_timer_start(sb_model *m, int32_t kernel_class, int32_t capacity);

/* Waits for the recorded events, returns the summed kernel time in
 * milliseconds and the number of timed launches, and releases the events. */
sb_status sb_timer_stop(sb_model *m, double *total_ms, int32_t *launches);

#ifdef __cplusplus
}
#endif

#endif /* SB_H */
