// C ABI of libsb: argument validation, workspace layout and the launch
// sequence of the verify step.  Every check runs on the host before anything
// is enqueued; the device work is in k_*.hip.
#include <math.h>
#include <string.h>

#include <mutex>
#include <new>
#include <vector>

#include "sb_internal_fwd.h"

struct sb_timer {
  int active = 0;
  int kernel_class = -1;
  int used = 0;
  std::vector<hipEvent_t> start, stop;
};

struct sb_model {
  sb_model_config cfg;
  std::vector<sb_layer_weights> layers;
  const void *embed;
  const float *final_norm;
  const void *lm_head;
  sb_timer timer;
  // H-RAD feature tap: residual after each of the last tap_k layers,
  // [tap_k][tap_rows][hidden] fp32 (null: no tap)
  float *tap = nullptr;
  int tap_k = 0, tap_rows = 0;
  int fwd_mode = SB_FWD_AUTO;  // sb_model_set_forward
};

// Scratch memory of sb_verify_forward_noalloc: the forward's workspace as a
// file-scope device array, one copy per device the library runs on, held
// until the process ends.  Host code never passes this name to a kernel:
// it is a host-side stand-in; the device address comes from
// hipGetSymbolAddress, once per device.
static __device__ __align__(256) char scratch[SB_NOALLOC_SCRATCH_BYTES];

namespace sb {
thread_local LaunchEvents g_launch_events;
namespace {

constexpr size_t kAlign = 256;
constexpr int kF32MaxKeys = 15360;  // scores of one row in 60 KB of LDS
constexpr int kBf16MaxKeys = 65536;  // cache slots a bf16 step may attend to

inline size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

struct Layout {
  size_t meta, rope, h, delta;
  // bf16
  size_t xa, act, q, part_o, part_ml, xn, ss, rs, pk_table, pk_sync;
  // f32
  size_t fa, qkv, fq, fo, gu, fact;
  size_t total;
  int np, n_chunks, pk_chunks, ks_h, ks_o, ks_f;
};

// Compute units of the current device (256 when it cannot be queried: the
// layout must not depend on a device being present).
int device_cus_host() {
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
      cus <= 0)
    return 256;
  return cus;
}

Layout make_layout(const sb_model_config &c, int n_rows, int kv_len) {
  Layout L{};
  const int np = round_up(n_rows, 16);
  const int H = c.hidden, d = c.head_dim, F = c.ffn;
  const int qd = c.n_heads * d, kvd = c.n_kv_heads * d;
  const int G = c.n_heads / c.n_kv_heads;
  L.np = np;
  size_t off = 0;
  auto take = [&](size_t bytes) {
    size_t o = off;
    off = align_up(off + bytes);
    return o;
  };
  L.meta = take(sizeof(Meta));
  L.rope = take((size_t)np * (d / 2) * sizeof(float2));
  L.h = take((size_t)np * H * sizeof(float));
  if (c.dtype == SB_BF16) {
    L.delta = take((size_t)kMaxSplit * np * H * sizeof(float));
    // packed activations use the k-steps of the weights they multiply
    L.ks_h = pack_geom(c, SB_W_QKV).ks;
    L.ks_o = pack_geom(c, SB_W_O).ks;
    L.ks_f = pack_geom(c, SB_W_DOWN).ks;
    const int ksx = L.ks_h > L.ks_o ? L.ks_h : L.ks_o;
    L.n_chunks = attn_splits(c.n_kv_heads, c.head_dim, kv_len + n_rows, n_rows * G);
    // key ranges of the persistent kernel's attention (one item per unit)
    L.pk_chunks = pk_attn_chunks(c.n_kv_heads, kv_len + n_rows, device_cus_host());
    const int chunks = L.n_chunks > L.pk_chunks ? L.n_chunks : L.pk_chunks;
    L.xa = take((size_t)np * ksx * 32 * 2);
    L.act = take((size_t)np * L.ks_f * 32 * 2);
    // the post-attention RMSNorm fused into the O projection: gated
    // residual (packed) and per-(token, group) sums of squares
    L.xn = take((size_t)np * L.ks_h * 32 * 2);
    L.ss = take((size_t)np * kSsGroups * sizeof(float));
    // 1/rms per row of the last RMSNorm kernel (its projection's scale)
    L.rs = take((size_t)np * sizeof(float));
    L.q = take((size_t)np * qd * 2);
    L.part_o = take((size_t)c.n_kv_heads * chunks * n_rows * G * d * sizeof(float));
    L.part_ml = take((size_t)c.n_kv_heads * chunks * n_rows * G * 2 * sizeof(float));
    // the persistent kernel's layer table and barrier counters
    L.pk_table = take((size_t)c.n_layers * sizeof(PkLayer));
    L.pk_sync = take(sizeof(PkSync));
  } else {
    L.fa = take((size_t)np * H * sizeof(float));
    L.qkv = take((size_t)np * (qd + 2 * kvd) * sizeof(float));
    L.fq = take((size_t)np * qd * sizeof(float));
    L.fo = take((size_t)np * qd * sizeof(float));
    L.gu = take((size_t)np * 2 * F * sizeof(float));
    L.fact = take((size_t)np * F * sizeof(float));
  }
  L.total = off;
  return L;
}

bool config_ok(const sb_model_config *c) {
  if (!c) return false;
  if (c->n_layers <= 0 || c->hidden <= 0 || c->n_heads <= 0 || c->n_kv_heads <= 0 ||
      c->head_dim <= 0 || c->ffn <= 0 || c->vocab <= 0)
    return false;
  if (c->n_heads % c->n_kv_heads != 0) return false;
  if (c->head_dim % 16 != 0) return false;
  if (!(c->rms_eps > 0.0f) || !(c->rope_theta > 0.0f)) return false;
  if (c->dtype != SB_F32 && c->dtype != SB_BF16) return false;
  return true;
}

sb_status shape_supported(const sb_model_config *c) {
  if (c->dtype == SB_BF16) {
    if (c->head_dim != 64 && c->head_dim != 128) return SB_ERR_UNSUPPORTED;
    if (c->hidden % 8 != 0 || c->hidden > 16384) return SB_ERR_UNSUPPORTED;
  } else {
    if (c->head_dim > 256) return SB_ERR_UNSUPPORTED;
  }
  return SB_OK;
}

sb_status check_tree(const int32_t *parents, int n, TreeArg *out) {
  if (!parents) return SB_ERR_INVALID_ARG;
  if (n < 1 || n > SB_MAX_ROWS) return SB_ERR_INVALID_ARG;
  if (parents[0] != -1) return SB_ERR_TREE;
  for (int i = 1; i < n; ++i)
    if (parents[i] < 0 || parents[i] >= i) return SB_ERR_TREE;
  if (out) {
    memset(out, 0, sizeof(*out));
    out->n = n;
    for (int i = 0; i < n; ++i) out->parent[i] = (int16_t)parents[i];
    for (int i = n; i < SB_MAX_ROWS; ++i) out->parent[i] = -2;  // no row
  }
  return SB_OK;
}

inline sb_status hip_status(hipError_t e) { return e == hipSuccess ? SB_OK : SB_ERR_HIP; }

#define SB_TRY(expr)                              \
  do {                                            \
    hipError_t _e = (expr);                       \
    if (_e != hipSuccess) return SB_ERR_HIP;      \
  } while (0)

size_t elem_bytes(const sb_model_config &c) { return c.dtype == SB_BF16 ? 2 : 4; }

// Embedding / metadata arguments, with the RoPE frequencies theta_j =
// base^(-2j/d) evaluated once on the host in float64.
EmbedArgs embed_args(const sb_model *m, const int32_t *tokens, float *h, int n, int kv_len,
                     Meta *meta, float2 *rope) {
  const sb_model_config &c = m->cfg;
  EmbedArgs ea{};
  ea.tokens = tokens;
  ea.embed = m->embed;
  ea.h = h;
  ea.vocab = c.vocab;
  ea.hidden = c.hidden;
  ea.n_tok = n;
  ea.kv_len = kv_len;
  ea.meta = meta;
  ea.rope = rope;
  ea.head_dim = c.head_dim;
  for (int j = 0; j < c.head_dim / 2 && j < 128; ++j)
    ea.theta[j] = pow((double)c.rope_theta, -2.0 * (double)j / (double)c.head_dim);
  return ea;
}

// Times one launch of kernel class kc with the model's timer events: a GEMM
// class hands them to its dispatch (which records the kernel's own start and
// end), any other class records them before and after its launch.
struct TimedLaunch {
  sb_timer &t;
  hipStream_t s;
  bool on, gemm;
  TimedLaunch(sb_model *m, int kc, hipStream_t st)
      : t(m->timer), s(st), on(m->timer.active && m->timer.kernel_class == kc &&
                               m->timer.used < (int)m->timer.start.size()),
        gemm(kc == SB_KC_QKV || kc == SB_KC_O || kc == SB_KC_GATE_UP || kc == SB_KC_DOWN ||
             kc == SB_KC_LM_HEAD) {
    if (!on) return;
    if (gemm)
      g_launch_events = LaunchEvents{t.start[t.used], t.stop[t.used], false};
    else
      (void)hipEventRecord(t.start[t.used], s);  // timing only: a failure costs a figure
  }
  ~TimedLaunch() {
    if (!on) return;
    if (!gemm) (void)hipEventRecord(t.stop[t.used], s);
    g_launch_events.taken = true;
    ++t.used;
  }
};

#define SB_TIMED(kc, expr)          \
  do {                              \
    TimedLaunch _tl(m, (kc), s);    \
    SB_TRY(expr);                   \
  } while (0)

sb_status forward_bf16(sb_model *m, const sb_kv_cache *kv, int kv_len, const int32_t *tokens,
                       const TreeArg &tree, int n, float temperature, float *logits,
                       sb_row_stats *stats, char *ws, const Layout &L, hipStream_t s) {
  const sb_model_config &c = m->cfg;
  const int H = c.hidden, d = c.head_dim;
  Meta *meta = (Meta *)(ws + L.meta);
  float2 *rope = (float2 *)(ws + L.rope);
  float *h = (float *)(ws + L.h);
  float *delta = (float *)(ws + L.delta);
  uint16_t *xa = (uint16_t *)(ws + L.xa);
  uint16_t *act = (uint16_t *)(ws + L.act);
  uint16_t *q = (uint16_t *)(ws + L.q);
  uint16_t *xn = (uint16_t *)(ws + L.xn);
  float *ss = (float *)(ws + L.ss);
  float *rs = (float *)(ws + L.rs);

  EmbedArgs ea = embed_args(m, tokens, h, n, kv_len, meta, rope);
  SB_TRY(launch_embed_meta(ea, tree, L.np, 1, s));

  const PackGeom gq = pack_geom(c, SB_W_QKV), go = pack_geom(c, SB_W_O),
                 gg = pack_geom(c, SB_W_GATE_UP), gd = pack_geom(c, SB_W_DOWN),
                 gl = pack_geom(c, SB_W_LM_HEAD);
  const size_t layer_kv = (size_t)c.n_kv_heads * kv->capacity * d;

  GemmArgs ga{};
  ga.n_tok = n;
  ga.q = q;
  ga.cap = kv->capacity;
  ga.kv_len = kv_len;
  ga.n_heads = c.n_heads;
  ga.n_kv = c.n_kv_heads;
  ga.head_dim = d;
  ga.rope = rope;
  ga.h = delta;
  ga.act = act;
  ga.act_ks = L.ks_f;
  ga.logits = logits;

  AttnArgs aa{};
  aa.q = q;
  aa.cap = kv->capacity;
  aa.kv_len = kv_len;
  aa.n_tok = n;
  aa.n_heads = c.n_heads;
  aa.n_kv = c.n_kv_heads;
  aa.head_dim = d;
  aa.n_chunks = L.n_chunks;
  aa.meta = meta;
  aa.scale = 1.0f / sqrtf((float)d);
  aa.part_o = (float *)(ws + L.part_o);
  aa.part_ml = (float *)(ws + L.part_ml);

  // H-RAD tap: the norm that adds layer li's output to the residual also
  // copies it when li is one of the last tap_k layers
  auto tap_of = [&](int li) -> float * {
    const int idx = li - (c.n_layers - m->tap_k);
    if (!m->tap || li < 0 || idx < 0) return nullptr;
    return m->tap + (size_t)idx * m->tap_rows * H;
  };

  // The O projection also applies the post-attention RMSNorm when its
  // launch shape allows (RESID_NORM); gate/up then scales by 1 / rms.
  int o_groups = 0;
  const bool fuse_norm = resid_norm_fusable(go.tiles, go.ks, n, &o_groups);
  int split = 0;  // delta slices left by the last residual projection
  for (int l = 0; l < c.n_layers; ++l) {
    const sb_layer_weights &lw = m->layers[l];
    uint16_t *kc = (uint16_t *)kv->k + l * layer_kv;
    uint16_t *vc = (uint16_t *)kv->v + l * layer_kv;
    SB_TIMED(SB_KC_NORM, launch_rmsnorm_pack(h, split ? delta : nullptr, split ? split : 1,
                                             lw.attn_norm, H, L.ks_h, n, L.np, c.rms_eps, xa, rs,
                                             s, tap_of(l - 1)));
    ga.W = (const uint16_t *)lw.qkv;
    ga.X = xa;
    ga.ks = gq.ks;
    ga.rs_in = rs;
    ga.kc = kc;
    ga.vc = vc;
    SB_TIMED(SB_KC_QKV, launch_gemm(EPI_QKV, ga, gq.tiles, nullptr, s));
    aa.kc = kc;
    aa.vc = vc;
    SB_TIMED(SB_KC_ATTN, launch_attn_bf16(aa, s));
    SB_TIMED(SB_KC_ATTN_MERGE, launch_attn_merge_bf16(aa, xa, L.ks_o, s));
    ga.W = (const uint16_t *)lw.o;
    ga.X = xa;
    ga.ks = go.ks;
    ga.out_rows = H;
    if (fuse_norm) {
      GemmArgs gn = ga;
      gn.h = h;
      gn.gain = lw.mlp_norm;
      gn.xn = xn;
      gn.xn_ks = L.ks_h;
      gn.ss = ss;
      gn.rs_in = nullptr;
      SB_TIMED(SB_KC_O, launch_gemm(EPI_RESID_NORM, gn, go.tiles, nullptr, s));
      ga.X = xn;
      ga.ss_in = ss;
      ga.ss_groups = o_groups;
      ga.norm_dim = H;
      ga.eps = c.rms_eps;
    } else {
      ga.rs_in = nullptr;
      SB_TIMED(SB_KC_O, launch_gemm(EPI_RESID, ga, go.tiles, &split, s));
      SB_TIMED(SB_KC_NORM, launch_rmsnorm_pack(h, delta, split, lw.mlp_norm, H, L.ks_h, n, L.np,
                                               c.rms_eps, xa, rs, s));
      ga.X = xa;
      ga.rs_in = rs;
    }
    ga.W = (const uint16_t *)lw.gate_up;
    ga.ks = gg.ks;
    SB_TIMED(SB_KC_GATE_UP, launch_gemm(EPI_SWIGLU, ga, gg.tiles, nullptr, s));
    ga.ss_in = nullptr;
    ga.rs_in = nullptr;
    ga.W = (const uint16_t *)lw.down;
    ga.X = act;
    ga.ks = gd.ks;
    ga.out_rows = H;
    SB_TIMED(SB_KC_DOWN, launch_gemm(EPI_RESID, ga, gd.tiles, &split, s));
  }
  // the last layer's H-RAD state is the final norm's output
  SB_TIMED(SB_KC_NORM, launch_rmsnorm_pack(h, split ? delta : nullptr, split ? split : 1,
                                           m->final_norm, H, L.ks_h, n, L.np, c.rms_eps, xa, rs,
                                           s, tap_of(c.n_layers - 1), 1));
  ga.W = (const uint16_t *)m->lm_head;
  ga.rs_in = rs;
  ga.X = xa;
  ga.ks = gl.ks;
  ga.out_rows = c.vocab;
  // The row softmax statistics come out of the LM head's epilogue as
  // per-(row, workgroup) partials, kept in the delta buffer (free once the
  // final norm has summed it), and one short pass combines them; the
  // logits are not read again.  Shapes whose partials do not fit there, and
  // trees of more than 128 rows (the LM head in k_gemm_wide), run the
  // statistics pass over the logits.
  const GemmPlan lp = plan_gemm(EPI_LOGITS, gl.tiles, gl.ks, n);
  const bool fuse_stats = !lp.wide && lp.groups <= kSsGroups &&
                          (size_t)n * lp.groups * sizeof(LmPart) <=
                              (size_t)kMaxSplit * L.np * H * sizeof(float);
  if (fuse_stats) {
    ga.lm_part = (LmPart *)delta;
    ga.lm_greedy = temperature <= 0.0f ? 1 : 0;
    ga.lm_inv_t = ga.lm_greedy ? 1.0f : 1.0f / temperature;
  }
  SB_TIMED(SB_KC_LM_HEAD, launch_gemm(EPI_LOGITS, ga, gl.tiles, nullptr, s));
  if (fuse_stats)
    SB_TIMED(SB_KC_STATS, launch_stats_finish((const LmPart *)delta, lp.groups, n, temperature,
                                              stats, s));
  else
    SB_TIMED(SB_KC_STATS, launch_softmax_stats(c.vocab, n, logits, temperature, stats, s));
  return SB_OK;
}

// The persistent forward of a bf16 model: embedding and tree metadata, the
// layer table, one cooperative launch for every layer and the LM head, then
// the row statistics.
sb_status forward_persist(sb_model *m, const sb_kv_cache *kv, int kv_len, const int32_t *tokens,
                          const TreeArg &tree, int n, float temperature, float *logits,
                          sb_row_stats *stats, char *ws, const Layout &L, PkArgs &a,
                          const void *kernel, int nwg, hipStream_t s) {
  const sb_model_config &c = m->cfg;
  Meta *meta = (Meta *)(ws + L.meta);
  float2 *rope = (float2 *)(ws + L.rope);
  float *h = (float *)(ws + L.h);
  EmbedArgs ea = embed_args(m, tokens, h, n, kv_len, meta, rope);
  SB_TRY(launch_embed_meta(ea, tree, L.np, 1, s));
  PkLayer *table = (PkLayer *)(ws + L.pk_table);
  for (int l0 = 0; l0 < c.n_layers; l0 += kPkTableLayers) {
    PkTableArgs t{};
    t.n = c.n_layers - l0 < kPkTableLayers ? c.n_layers - l0 : kPkTableLayers;
    for (int i = 0; i < t.n; ++i) {
      const sb_layer_weights &lw = m->layers[l0 + i];
      t.layer[i] = PkLayer{(const uint16_t *)lw.qkv, (const uint16_t *)lw.o,
                           (const uint16_t *)lw.gate_up, (const uint16_t *)lw.down,
                           lw.attn_norm, lw.mlp_norm};
    }
    t.dst = table + l0;
    t.sync = l0 == 0 ? (PkSync *)(ws + L.pk_sync) : nullptr;
    SB_TRY(launch_pk_table(t, s));
  }
  a.n_tok = n;
  a.kv_len = kv_len;
  a.cap = kv->capacity;
  a.n_chunks = L.pk_chunks;
  a.layers = table;
  a.lm_head = (const uint16_t *)m->lm_head;
  a.g_final = m->final_norm;
  a.kc = (uint16_t *)kv->k;
  a.vc = (uint16_t *)kv->v;
  a.layer_kv = (size_t)c.n_kv_heads * kv->capacity * c.head_dim;
  a.h = h;
  a.delta = (float *)(ws + L.delta);
  a.ss = (float *)(ws + L.ss);
  a.part_o = (float *)(ws + L.part_o);
  a.part_ml = (float *)(ws + L.part_ml);
  a.logits = logits;
  a.xa = (uint16_t *)(ws + L.xa);
  a.xo = (uint16_t *)(ws + L.xa);  // the attention output reuses the norm's buffer
  a.act = (uint16_t *)(ws + L.act);
  a.q = (uint16_t *)(ws + L.q);
  a.meta = meta;
  a.rope = rope;
  a.sync = (PkSync *)(ws + L.pk_sync);
  SB_TIMED(SB_KC_PERSIST, launch_persist(a, kernel, nwg, s));
  SB_TIMED(SB_KC_STATS, launch_softmax_stats(c.vocab, n, logits, temperature, stats, s,
                                             &a.sync->status[0]));
  return SB_OK;
}

sb_status forward_f32(sb_model *m, const sb_kv_cache *kv, int kv_len, const int32_t *tokens,
                      const TreeArg &tree, int n, float temperature, float *logits,
                      sb_row_stats *stats, char *ws, const Layout &L, hipStream_t s) {
  const sb_model_config &c = m->cfg;
  const int H = c.hidden, d = c.head_dim, F = c.ffn;
  const int qd = c.n_heads * d, kvd = c.n_kv_heads * d;
  Meta *meta = (Meta *)(ws + L.meta);
  float2 *rope = (float2 *)(ws + L.rope);
  float *h = (float *)(ws + L.h);
  float *a = (float *)(ws + L.fa);
  float *qkv = (float *)(ws + L.qkv);
  float *q = (float *)(ws + L.fq);
  float *o = (float *)(ws + L.fo);
  float *gu = (float *)(ws + L.gu);
  float *act = (float *)(ws + L.fact);

  EmbedArgs ea = embed_args(m, tokens, h, n, kv_len, meta, rope);
  SB_TRY(launch_embed_meta(ea, tree, n, 0, s));
  const size_t layer_kv = (size_t)c.n_kv_heads * kv->capacity * d;

  AttnArgs aa{};
  aa.q = q;
  aa.cap = kv->capacity;
  aa.kv_len = kv_len;
  aa.n_tok = n;
  aa.n_heads = c.n_heads;
  aa.n_kv = c.n_kv_heads;
  aa.head_dim = d;
  aa.meta = meta;
  aa.scale = 1.0f / sqrtf((float)d);

  for (int l = 0; l < c.n_layers; ++l) {
    const sb_layer_weights &lw = m->layers[l];
    float *kc = (float *)kv->k + l * layer_kv;
    float *vc = (float *)kv->v + l * layer_kv;
    SB_TRY(launch_f32_rmsnorm(h, lw.attn_norm, H, n, c.rms_eps, a, s));
    SB_TRY(launch_f32_gemm(a, (const float *)lw.qkv, qkv, n, qd + 2 * kvd, H, qd + 2 * kvd, 0, s));
    SB_TRY(launch_f32_rope_qkv(qkv, c, n, rope, q, kc, vc, kv->capacity, kv_len, s));
    aa.kc = kc;
    aa.vc = vc;
    SB_TRY(launch_f32_attn(aa, o, s));
    SB_TRY(launch_f32_gemm(o, (const float *)lw.o, h, n, H, qd, H, 1, s));
    SB_TRY(launch_f32_rmsnorm(h, lw.mlp_norm, H, n, c.rms_eps, a, s));
    SB_TRY(launch_f32_gemm(a, (const float *)lw.gate_up, gu, n, 2 * F, H, 2 * F, 0, s));
    SB_TRY(launch_f32_swiglu(gu, n, F, act, s));
    SB_TRY(launch_f32_gemm(act, (const float *)lw.down, h, n, H, F, H, 1, s));
  }
  SB_TRY(launch_f32_rmsnorm(h, m->final_norm, H, n, c.rms_eps, a, s));
  SB_TRY(launch_f32_gemm(a, (const float *)m->lm_head, logits, n, c.vocab, H, c.vocab, 0, s));
  SB_TRY(launch_softmax_stats(c.vocab, n, logits, temperature, stats, s));
  return SB_OK;
}

bool temperature_ok(float t) { return isfinite(t) && t >= 0.0f; }

}  // namespace

bool pk_plan(const sb_model_config &c, int n_tok, int nwg, PkArgs *a, const void **kernel) {
  if (c.dtype != SB_BF16 || c.head_dim != 128 || c.n_heads % c.n_kv_heads != 0) return false;
  if (n_tok < 1 || n_tok > 64 || nwg < 8 || nwg > kSsGroups) return false;
  const int tt = (n_tok + 15) / 16;
  const int G = c.n_heads / c.n_kv_heads;
  const int rt = G == 1 ? tt : 4;  // grouped queries: 64-row attention blocks
  // the norm phase: 8-column groups of the packed width over the units, at
  // most 8 per unit and one thread per (row, group)
  const int ks_h = pack_geom(c, SB_W_QKV).ks;
  const int gpw = (ks_h * 4 + nwg - 1) / nwg;
  if (gpw > 8 || gpw * n_tok > kPkThreadsHost) return false;
  PkArgs p{};
  p.n_layers = c.n_layers;
  p.hidden = c.hidden;
  p.n_heads = c.n_heads;
  p.n_kv = c.n_kv_heads;
  p.head_dim = c.head_dim;
  p.ffn = c.ffn;
  p.vocab = c.vocab;
  p.eps = c.rms_eps;
  p.scale = 1.0f / sqrtf((float)c.head_dim);
  p.xa_ks = ks_h;
  p.xo_ks = pack_geom(c, SB_W_O).ks;
  p.act_ks = pack_geom(c, SB_W_DOWN).ks;
  struct K {
    int kind, epi;
    PkGemmPlan *dst;
  } kinds[] = {{SB_W_QKV, EPI_QKV, &p.qkv},
               {SB_W_O, EPI_RESID, &p.o},
               {SB_W_GATE_UP, EPI_SWIGLU, &p.gu},
               {SB_W_DOWN, EPI_RESID, &p.dn},
               {SB_W_LM_HEAD, EPI_LOGITS, &p.lm}};
  // the planner's tiles per pass, and whether they are the special set
  // (3 / 4 / 6 / 4 / 8 at three token tiles); otherwise the generic set
  // 4 / 4 / 8 / 4 / 8 (passes as many as a group's tiles need)
  static const int special[5] = {3, 4, 6, 4, 8}, generic[5] = {4, 4, 8, 4, 8};
  bool is_special = tt == 3 && rt == 3;
  GemmPlan gp[5];
  for (int i = 0; i < 5; ++i) {
    const PackGeom g = pack_geom(c, kinds[i].kind);
    gp[i] = plan_gemm(kinds[i].epi, g.tiles, g.ks, n_tok);
    if (gp[i].tt != tt || gp[i].split > kMaxSplit || gp[i].grid > nwg) return false;
    if (gp[i].nt != special[i]) is_special = false;
  }
  for (int i = 0; i < 5; ++i) {
    const PackGeom g = pack_geom(c, kinds[i].kind);
    *kinds[i].dst = PkGemmPlan{g.ks, g.tiles, is_special ? special[i] : generic[i], gp[i].split,
                               gp[i].groups};
  }
  const void *k = pk_kernel(tt, rt, is_special);
  if (!k) return false;
  *a = p;
  *kernel = k;
  return true;
}

}  // namespace sb

using namespace sb;

extern "C" {

const char *sb_status_string(sb_status st) {
  switch (st) {
    case SB_OK:
      return "ok";
    case SB_ERR_INVALID_ARG:
      return "invalid argument";
    case SB_ERR_TREE:
      return "parents do not form a rooted tree in row order";
    case SB_ERR_CAPACITY:
      return "KV capacity or workspace too small";
    case SB_ERR_DTYPE:
      return "dtype not supported for this call";
    case SB_ERR_HIP:
      return "HIP call or kernel launch failed";
    case SB_ERR_UNSUPPORTED:
      return "shape not supported by the kernels";
  }
  return "unknown status";
}

int32_t sb_version(void) { return 1; }

size_t sb_packed_bytes(const sb_model_config *cfg, int32_t kind) {
  if (!config_ok(cfg) || kind < SB_W_QKV || kind > SB_W_LM_HEAD) return 0;
  return pack_geom(*cfg, kind).bytes;
}

sb_status sb_pack_weight(const sb_model_config *cfg, int32_t kind, const void *src0,
                         const void *src1, const void *src2, void *dst, hipStream_t stream) {
  if (!config_ok(cfg) || kind < SB_W_QKV || kind > SB_W_LM_HEAD || !src0 || !dst)
    return SB_ERR_INVALID_ARG;
  if ((kind == SB_W_QKV && (!src1 || !src2)) || (kind == SB_W_GATE_UP && !src1))
    return SB_ERR_INVALID_ARG;
  const sb_model_config &c = *cfg;
  if (c.dtype == SB_BF16) {
    if (shape_supported(cfg) != SB_OK) return SB_ERR_UNSUPPORTED;
    return hip_status(launch_pack_bf16(kind, c, src0, src1, src2, dst, stream));
  }
  // float32: concatenated row-major sources
  const size_t H = c.hidden, qd = (size_t)c.n_heads * c.head_dim,
               kvd = (size_t)c.n_kv_heads * c.head_dim, F = c.ffn;
  char *o = (char *)dst;
  auto cp = [&](const void *src, size_t bytes) -> hipError_t {
    hipError_t e = hipMemcpyAsync(o, src, bytes, hipMemcpyDeviceToDevice, stream);
    o += bytes;
    return e;
  };
  hipError_t e = hipSuccess;
  switch (kind) {
    case SB_W_QKV:
      if ((e = cp(src0, qd * H * 4)) != hipSuccess) break;
      if ((e = cp(src1, kvd * H * 4)) != hipSuccess) break;
      e = cp(src2, kvd * H * 4);
      break;
    case SB_W_O:
      e = cp(src0, H * qd * 4);
      break;
    case SB_W_GATE_UP:
      if ((e = cp(src0, F * H * 4)) != hipSuccess) break;
      e = cp(src1, F * H * 4);
      break;
    case SB_W_DOWN:
      e = cp(src0, H * F * 4);
      break;
    case SB_W_LM_HEAD:
      e = cp(src0, (size_t)c.vocab * H * 4);
      break;
  }
  return hip_status(e);
}

sb_status sb_model_create(const sb_model_config *cfg, const sb_model_weights *w, sb_model **out) {
  if (!out) return SB_ERR_INVALID_ARG;
  *out = nullptr;
  if (!config_ok(cfg) || !w) return SB_ERR_INVALID_ARG;
  sb_status st = shape_supported(cfg);
  if (st != SB_OK) return st;
  if (!w->embed || !w->final_norm || !w->lm_head || !w->layers) return SB_ERR_INVALID_ARG;
  for (int l = 0; l < cfg->n_layers; ++l) {
    const sb_layer_weights &lw = w->layers[l];
    if (!lw.attn_norm || !lw.qkv || !lw.o || !lw.mlp_norm || !lw.gate_up || !lw.down)
      return SB_ERR_INVALID_ARG;
  }
  sb_model *m = new (std::nothrow) sb_model;
  if (!m) return SB_ERR_INVALID_ARG;
  m->cfg = *cfg;
  m->layers.assign(w->layers, w->layers + cfg->n_layers);
  m->embed = w->embed;
  m->final_norm = w->final_norm;
  m->lm_head = w->lm_head;
  *out = m;
  return SB_OK;
}

static void timer_release(sb_timer &t) {
  for (hipEvent_t e : t.start) (void)hipEventDestroy(e);
  for (hipEvent_t e : t.stop) (void)hipEventDestroy(e);
  t.start.clear();
  t.stop.clear();
  t.active = 0;
  t.used = 0;
}

void sb_model_destroy(sb_model *m) {
  if (!m) return;
  timer_release(m->timer);
  delete m;
}

sb_status sb_timer_start(sb_model *m, int32_t kernel_class, int32_t capacity) {
  if (!m || kernel_class < SB_KC_QKV || kernel_class > SB_KC_PERSIST || capacity < 1 ||
      capacity > (1 << 20))
    return SB_ERR_INVALID_ARG;
  timer_release(m->timer);
  sb_timer &t = m->timer;
  t.start.resize(capacity);
  t.stop.resize(capacity);
  for (int i = 0; i < capacity; ++i) {
    if (hipEventCreate(&t.start[i]) != hipSuccess || hipEventCreate(&t.stop[i]) != hipSuccess) {
      t.start.resize(i);
      t.stop.resize(i);
      timer_release(t);
      return SB_ERR_HIP;
    }
  }
  t.kernel_class = kernel_class;
  t.used = 0;
  t.active = 1;
  return SB_OK;
}

sb_status sb_timer_stop(sb_model *m, double *total_ms, int32_t *launches) {
  if (!m || !total_ms || !launches) return SB_ERR_INVALID_ARG;
  sb_timer &t = m->timer;
  double sum = 0.0;
  sb_status st = SB_OK;
  for (int i = 0; i < t.used; ++i) {
    float ms = 0.0f;
    if (hipEventSynchronize(t.stop[i]) != hipSuccess ||
        hipEventElapsedTime(&ms, t.start[i], t.stop[i]) != hipSuccess) {
      st = SB_ERR_HIP;
      break;
    }
    sum += ms;
  }
  *total_ms = sum;
  *launches = t.used;
  timer_release(t);
  return st;
}

size_t sb_workspace_bytes(const sb_model *m, int32_t max_rows, int32_t max_kv_len) {
  if (!m || max_rows < 1 || max_rows > SB_MAX_ROWS || max_kv_len < 0) return 0;
  return make_layout(m->cfg, max_rows, max_kv_len).total;
}

sb_status sb_verify_forward(sb_model *m, const sb_kv_cache *kv, int32_t kv_len,
                            const int32_t *d_tokens, const int32_t *h_parents, int32_t n_rows,
                            float temperature, float *d_logits, sb_row_stats *d_stats,
                            void *d_ws, size_t ws_bytes, hipStream_t stream) {
  if (!m || !kv || !kv->k || !kv->v || !d_tokens || !d_logits || !d_stats || !d_ws)
    return SB_ERR_INVALID_ARG;
  if (kv_len < 0 || !temperature_ok(temperature)) return SB_ERR_INVALID_ARG;
  TreeArg tree;
  sb_status st = check_tree(h_parents, n_rows, &tree);
  if (st != SB_OK) return st;
  if ((int64_t)kv_len + n_rows > kv->capacity || kv->capacity % 8 != 0) return SB_ERR_CAPACITY;
  if (m->cfg.dtype == SB_BF16 && (int64_t)kv_len + n_rows > kBf16MaxKeys) return SB_ERR_UNSUPPORTED;
  if (m->cfg.dtype == SB_F32 && kv_len + n_rows > kF32MaxKeys) return SB_ERR_UNSUPPORTED;
  const Layout L = make_layout(m->cfg, n_rows, kv_len);
  if (ws_bytes < L.total) return SB_ERR_CAPACITY;
  if (m->tap && n_rows > m->tap_rows) return SB_ERR_CAPACITY;
  if (m->cfg.dtype == SB_BF16) {
    // the persistent forward only when asked for (it measured slower than
    // the chain: a device-wide barrier costs about what a launch does), and
    // not with the H-RAD tap (the chain writes it)
    if (m->fwd_mode == SB_FWD_PERSISTENT && !m->tap) {
      PkArgs a;
      const void *kernel = nullptr;
      const int nwg = device_cus_host();
      if (pk_plan(m->cfg, n_rows, nwg, &a, &kernel))
        return forward_persist(m, kv, kv_len, d_tokens, tree, n_rows, temperature, d_logits,
                               d_stats, (char *)d_ws, L, a, kernel, nwg, stream);
    }
    if (m->fwd_mode == SB_FWD_PERSISTENT) return SB_ERR_UNSUPPORTED;
    return forward_bf16(m, kv, kv_len, d_tokens, tree, n_rows, temperature, d_logits, d_stats,
                        (char *)d_ws, L, stream);
  }
  if (m->fwd_mode == SB_FWD_PERSISTENT) return SB_ERR_UNSUPPORTED;
  return forward_f32(m, kv, kv_len, d_tokens, tree, n_rows, temperature, d_logits, d_stats,
                     (char *)d_ws, L, stream);
}

// Device address of this device's scratch array, looked up once per device
// (with that device current) and kept.
static sb_status scratch_address(void **out) {
  static std::mutex mu;
  static void *addr[SB_NOALLOC_MAX_DEVICES] = {};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= SB_NOALLOC_MAX_DEVICES)
    return SB_ERR_HIP;
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[dev]) {
    void *p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return SB_ERR_HIP;
    addr[dev] = p;
  }
  *out = addr[dev];
  return SB_OK;
}

sb_status sb_verify_forward_noalloc(sb_model *m, const sb_kv_cache *kv, int32_t kv_len,
                                    const int32_t *d_tokens, const int32_t *h_parents,
                                    int32_t n_rows, float temperature, float *d_logits,
                                    sb_row_stats *d_stats, hipStream_t stream) {
  if (!m || kv_len < 0 || n_rows < 1 || n_rows > SB_MAX_ROWS) return SB_ERR_INVALID_ARG;
  // the step's workspace must fit the scratch array (checked before any
  // device call)
  if (make_layout(m->cfg, n_rows, kv_len).total > (size_t)SB_NOALLOC_SCRATCH_BYTES)
    return SB_ERR_CAPACITY;
  void *ws = nullptr;
  sb_status st = scratch_address(&ws);
  if (st != SB_OK) return st;
  return sb_verify_forward(m, kv, kv_len, d_tokens, h_parents, n_rows, temperature, d_logits,
                           d_stats, ws, (size_t)SB_NOALLOC_SCRATCH_BYTES, stream);
}

sb_status sb_softmax_stats(int32_t vocab, int32_t n_rows, const float *d_logits,
                           float temperature, sb_row_stats *d_stats, hipStream_t stream) {
  if (vocab < 1 || n_rows < 1 || !d_logits || !d_stats || !temperature_ok(temperature))
    return SB_ERR_INVALID_ARG;
  return hip_status(launch_softmax_stats(vocab, n_rows, d_logits, temperature, d_stats, stream));
}

size_t sb_sample_workspace_bytes(int32_t vocab) {
  if (vocab < 1) return 0;
  return sample_ws_bytes(vocab);
}

sb_status sb_select_branch(int32_t vocab, const float *d_logits_row,
                           const sb_row_stats *d_stats_row, float temperature, int32_t n_cand,
                           const int32_t *d_cand_tokens, const float *d_q, const float *d_u,
                           int32_t *d_out, void *d_ws, size_t ws_bytes, hipStream_t stream) {
  if (vocab < 1 || !d_logits_row || !d_stats_row || !d_cand_tokens || !d_q || !d_u || !d_out ||
      !d_ws || !temperature_ok(temperature))
    return SB_ERR_INVALID_ARG;
  if (n_cand < 1 || n_cand > SB_MAX_ROWS) return SB_ERR_INVALID_ARG;
  if (ws_bytes < sample_ws_bytes(vocab)) return SB_ERR_CAPACITY;
  return hip_status(launch_select(vocab, d_logits_row, d_stats_row, temperature, n_cand,
                                  d_cand_tokens, d_q, d_u, d_out, d_ws, stream));
}

sb_status sb_accept_resample(int32_t vocab, int32_t n_rows, const int32_t *d_tokens,
                             const int32_t *h_parents, const float *d_logits,
                             const sb_row_stats *d_stats, float temperature, const float *d_q,
                             const float *d_u, sb_step_result *d_result, void *d_ws,
                             size_t ws_bytes, hipStream_t stream) {
  if (vocab < 1 || !d_tokens || !d_logits || !d_stats || !d_q || !d_u || !d_result || !d_ws ||
      !temperature_ok(temperature))
    return SB_ERR_INVALID_ARG;
  TreeArg tree;
  sb_status st = check_tree(h_parents, n_rows, &tree);
  if (st != SB_OK) return st;
  if (ws_bytes < sample_ws_bytes(vocab)) return SB_ERR_CAPACITY;
  return hip_status(launch_walk(vocab, tree, d_tokens, d_logits, d_stats, temperature, d_q, d_u,
                                d_result, d_ws, stream));
}

sb_status sb_model_set_forward(sb_model *m, int32_t mode) {
  if (!m || (mode != SB_FWD_AUTO && mode != SB_FWD_KERNELS && mode != SB_FWD_PERSISTENT))
    return SB_ERR_INVALID_ARG;
  m->fwd_mode = mode;
  return SB_OK;
}

sb_status sb_model_set_tap(sb_model *m, float *d_taps, int32_t k_layers, int32_t max_rows) {
  if (!m) return SB_ERR_INVALID_ARG;
  if (!d_taps) {
    m->tap = nullptr;
    m->tap_k = m->tap_rows = 0;
    return SB_OK;
  }
  if (m->cfg.dtype != SB_BF16) return SB_ERR_DTYPE;
  if (k_layers < 1 || k_layers > m->cfg.n_layers || max_rows < 1 || max_rows > SB_MAX_ROWS)
    return SB_ERR_INVALID_ARG;
  m->tap = d_taps;
  m->tap_k = k_layers;
  m->tap_rows = max_rows;
  return SB_OK;
}

size_t sb_hrad_workspace_bytes(void) { return align_up(SB_HRAD_H1 * sizeof(float)); }

sb_status sb_hrad_predict(const sb_model *m, const float *d_taps, int32_t k_layers,
                          int32_t max_rows, const sb_step_result *d_result,
                          const sb_hrad_weights *w, float *d_logits3, int32_t *d_class,
                          void *d_ws, size_t ws_bytes, hipStream_t stream) {
  if (!m || !d_taps || !d_result || !w || !d_logits3 || !d_class || !d_ws)
    return SB_ERR_INVALID_ARG;
  if (!w->w1 || !w->b1 || !w->w2 || !w->b2 || !w->w3 || !w->b3) return SB_ERR_INVALID_ARG;
  if (m->cfg.dtype != SB_BF16) return SB_ERR_DTYPE;
  if (k_layers < 1 || k_layers > m->cfg.n_layers || max_rows < 1 || max_rows > SB_MAX_ROWS)
    return SB_ERR_INVALID_ARG;
  if (ws_bytes < sb_hrad_workspace_bytes()) return SB_ERR_CAPACITY;
  HradArgs a{};
  a.taps = d_taps;
  a.k = k_layers;
  a.max_rows = max_rows;
  a.hidden = m->cfg.hidden;
  a.vocab = m->cfg.vocab;
  a.embed = (const uint16_t *)m->embed;
  a.res = d_result;
  a.w1 = w->w1;
  a.b1 = w->b1;
  a.w2 = w->w2;
  a.b2 = w->b2;
  a.w3 = w->w3;
  a.b3 = w->b3;
  a.y1 = (float *)d_ws;
  a.logits3 = d_logits3;
  a.cls = d_class;
  return hip_status(launch_hrad(a, stream));
}

size_t sb_branch_workspace_bytes(void) { return 256; }

sb_status sb_branch_candidates(const float *d_q, int32_t vocab, const int32_t *d_x_b, int32_t k_max,
                               int32_t mode, const float *d_u, int32_t *d_count,
                               int32_t *d_tokens, float *d_rows, void *d_ws, size_t ws_bytes,
                               hipStream_t stream) {
  if (!d_q || !d_x_b || !d_count || !d_tokens || !d_rows || !d_ws) return SB_ERR_INVALID_ARG;
  if (mode != SB_BRANCH_TOPK && mode != SB_BRANCH_IID && mode != SB_BRANCH_WOR)
    return SB_ERR_INVALID_ARG;
  if (mode != SB_BRANCH_TOPK && !d_u) return SB_ERR_INVALID_ARG;
  if (vocab < 1 || vocab > SB_BRANCH_MAX_VOCAB || k_max < 1 || k_max > SB_BRANCH_MAX_K)
    return SB_ERR_INVALID_ARG;
  if (ws_bytes < sb_branch_workspace_bytes()) return SB_ERR_CAPACITY;
  BranchArgs a{};
  a.q = d_q;
  a.vocab = vocab;
  a.x_b = d_x_b;
  a.k_max = k_max;
  a.mode = mode;
  a.vec4 = vocab % 4 == 0 && ((uintptr_t)d_q & 15) == 0 && ((uintptr_t)d_rows & 15) == 0;
  a.u = d_u;
  a.count = d_count;
  a.tokens = d_tokens;
  a.rows = d_rows;
  a.znorm = (double *)d_ws;
  return hip_status(launch_branch(a, stream));
}

sb_status sb_draft_sample(int32_t vocab, int32_t n, const float *d_logits,
                          const sb_row_stats *d_stats, int32_t n_logit_rows,
                          const int32_t *h_src_rows, float temperature, const float *d_u,
                          int32_t *d_tokens, float *d_q, int32_t n_out_rows,
                          const int32_t *h_dst_rows, void *d_ws, size_t ws_bytes,
                          hipStream_t stream) {
  if (!d_logits || !d_stats || !h_src_rows || !d_u || !d_tokens || !d_q || !h_dst_rows || !d_ws)
    return SB_ERR_INVALID_ARG;
  if (vocab < 1 || n < 1 || n > SB_DRAFT_MAX_ROWS || !temperature_ok(temperature))
    return SB_ERR_INVALID_ARG;
  if (ws_bytes < draft_ws_bytes(vocab, n)) return SB_ERR_CAPACITY;
  DraftRows rows{};
  rows.n = n;
  for (int i = 0; i < n; ++i) {
    if (h_src_rows[i] < 0 || h_src_rows[i] >= n_logit_rows) return SB_ERR_INVALID_ARG;
    if (h_dst_rows[i] < 0 || h_dst_rows[i] >= n_out_rows) return SB_ERR_INVALID_ARG;
    for (int j = 0; j < i; ++j)
      if (h_dst_rows[j] == h_dst_rows[i]) return SB_ERR_INVALID_ARG;
    rows.src[i] = h_src_rows[i];
    rows.dst[i] = h_dst_rows[i];
  }
  return hip_status(launch_draft_sample(vocab, rows, d_logits, d_stats, temperature, d_u, d_tokens,
                                       d_q, d_ws, stream));
}

size_t sb_draft_sample_workspace_bytes(int32_t vocab, int32_t n) {
  if (vocab < 1 || n < 1 || n > SB_DRAFT_MAX_ROWS) return 0;
  return draft_ws_bytes(vocab, n);
}

// Workspace of a draft round: the forward's, the logits and statistics of
// the largest tree, the candidates' and the sampler's workspaces, x_b, B and
// the drawn token's probability.
struct RoundLayout {
  size_t fwd, logits, stats, branch, sample, ints, total;
};
static bool round_layout(const sb_model *m, int k_max, int depth, int trunk_max, int kv_len,
                         RoundLayout *o) {
  if (!m || k_max < 1 || k_max > SB_BRANCH_MAX_K || depth < 1 || trunk_max < 1 || kv_len < 0)
    return false;
  if ((int64_t)trunk_max + (int64_t)k_max * depth > SB_MAX_ROWS) return false;
  const int R = trunk_max + k_max * depth;
  const size_t fw = sb_workspace_bytes(m, R, kv_len);
  if (!fw) return false;
  o->fwd = 0;
  o->logits = align_up(fw);
  o->stats = o->logits + align_up((size_t)R * m->cfg.vocab * 4);
  o->branch = o->stats + align_up((size_t)R * sizeof(sb_row_stats));
  o->sample = o->branch + align_up(sb_branch_workspace_bytes());
  o->ints = o->sample + align_up(draft_ws_bytes(m->cfg.vocab, k_max));
  o->total = o->ints + align_up(4 * sizeof(int32_t));
  return true;
}

size_t sb_draft_round_workspace_bytes(const sb_model *draft, int32_t k_max, int32_t depth,
                                      int32_t trunk_max, int32_t kv_len) {
  RoundLayout L;
  return round_layout(draft, k_max, depth, trunk_max, kv_len, &L) ? L.total : 0;
}

static bool draft_args_ok(sb_model *draft, const sb_kv_cache *kv, float temperature) {
  return draft && kv && kv->k && kv->v && temperature_ok(temperature) &&
         draft->cfg.vocab <= SB_BRANCH_MAX_VOCAB;
}

// Draws into logits rows of a drafting step (src -> dst rows of d_tokens /
// d_q), from the round workspace's logits and statistics.
static sb_status draft_sample_rows(const sb_model *draft, char *ws, const RoundLayout &L,
                                   float temperature, int n_logit_rows, int n, const int32_t *src,
                                   const int32_t *dst, int n_out, const float *u, int32_t *toks,
                                   float *d_q, float *cf, hipStream_t stream) {
  DraftRows rows{};
  rows.n = n;
  for (int i = 0; i < n; ++i) {
    if (src[i] < 0 || src[i] >= n_logit_rows || dst[i] < 0 || dst[i] >= n_out)
      return SB_ERR_INVALID_ARG;
    rows.src[i] = src[i];
    rows.dst[i] = dst[i];
  }
  return hip_status(launch_draft_sample(draft->cfg.vocab, rows, (const float *)(ws + L.logits),
                                        (const sb_row_stats *)(ws + L.stats), temperature, u,
                                        toks, d_q, ws + L.sample, stream, cf));
}

sb_status sb_draft_chain(sb_model *draft, const sb_kv_cache *kv, int32_t kv_len, int32_t trunk_max,
                         float confidence, int32_t flags, float temperature, const float *d_u,
                         int32_t *d_tokens, float *d_q, int32_t *d_xb, int32_t *h_chain,
                         void *d_ws, size_t ws_bytes, hipStream_t stream) {
  if (!draft_args_ok(draft, kv, temperature) || !d_u || !d_tokens || !d_q || !d_xb || !h_chain ||
      !d_ws || isnan(confidence) || (flags & ~SB_CHAIN_CONDITIONED) != 0)
    return SB_ERR_INVALID_ARG;
  RoundLayout L;
  if (!round_layout(draft, 1, 1, trunk_max, kv_len, &L)) return SB_ERR_INVALID_ARG;
  if (ws_bytes < L.total) return SB_ERR_CAPACITY;
  if ((int64_t)kv_len + trunk_max > kv->capacity) return SB_ERR_CAPACITY;
  const int V = draft->cfg.vocab;
  char *ws = (char *)d_ws;
  float *logits = (float *)(ws + L.logits);
  sb_row_stats *stats = (sb_row_stats *)(ws + L.stats);
  float *conf = (float *)((int32_t *)(ws + L.ints) + 2);
  const size_t fws = L.logits;
  // x_t from row t - 1, until the first token below the confidence
  // threshold or x_trunk_max, which becomes x_b
  int32_t par[SB_MAX_ROWS];
  par[0] = -1;
  for (int t = 1; t <= trunk_max; ++t) {
    sb_status st = sb_verify_forward(draft, kv, kv_len, d_tokens, par, t, temperature, logits,
                                     stats, ws, fws, stream);
    if (st != SB_OK) return st;
    const int32_t src = t - 1;
    if (t == trunk_max) {
      // the last allowed draft is the branch point: its row goes straight
      // to row 0, its token to x_b
      const int32_t zero = 0;
      st = draft_sample_rows(draft, ws, L, temperature, t, 1, &src, &zero, trunk_max + 1,
                             d_u + (t - 1), d_xb, d_q, nullptr, stream);
      if (st != SB_OK) return st;
      *h_chain = t - 1;
      return SB_OK;
    }
    const int32_t dst = t;
    st = draft_sample_rows(draft, ws, L, temperature, t, 1, &src, &dst, trunk_max + 1,
                           d_u + (t - 1), d_tokens, d_q, conf, stream);
    if (st != SB_OK) return st;
    // A probability is never below a threshold <= 0 (a NaN one is not below
    // any): then every draft is confident and the host reads nothing.
    float cf = 0.0f;
    if (confidence > 0.0f &&
        (hipMemcpyAsync(&cf, conf, sizeof(cf), hipMemcpyDeviceToHost, stream) != hipSuccess ||
         hipStreamSynchronize(stream) != hipSuccess))
      return SB_ERR_HIP;
    if (confidence > 0.0f && cf < confidence) {
      // an unconfident draft: the branch point; its distribution to row 0,
      // its token to x_b
      if (hipMemcpyAsync(d_q, d_q + (size_t)t * V, (size_t)V * sizeof(float),
                         hipMemcpyDeviceToDevice, stream) != hipSuccess ||
          hipMemcpyAsync(d_xb, d_tokens + t, sizeof(int32_t), hipMemcpyDeviceToDevice,
                         stream) != hipSuccess)
        return SB_ERR_HIP;
      *h_chain = t - 1;
      return SB_OK;
    }
    // a confident draft: with SB_CHAIN_CONDITIONED its row becomes q
    // conditioned on confidence, the row its test divides by
    if ((flags & SB_CHAIN_CONDITIONED) &&
        launch_confident_row(d_q + (size_t)t * V, V, confidence, stream) != hipSuccess)
      return SB_ERR_HIP;
    par[t] = t - 1;
  }
  return SB_ERR_INVALID_ARG;  // not reached: t == trunk_max returns
}

sb_status sb_draft_branches(sb_model *draft, const sb_kv_cache *kv, int32_t kv_len, int32_t chain,
                            const int32_t *d_xb, int32_t k_max, int32_t mode, int32_t depth,
                            float temperature, const float *d_u, int32_t *d_tokens, float *d_q,
                            int32_t *h_parents, int32_t *h_branches, void *d_ws, size_t ws_bytes,
                            hipStream_t stream) {
  if (!draft_args_ok(draft, kv, temperature) || !d_xb || !d_u || !d_tokens || !d_q ||
      !h_parents || !h_branches || !d_ws || chain < 0)
    return SB_ERR_INVALID_ARG;
  if (mode != SB_BRANCH_TOPK && mode != SB_BRANCH_IID && mode != SB_BRANCH_WOR)
    return SB_ERR_INVALID_ARG;
  RoundLayout L;
  if (!round_layout(draft, k_max, depth, chain + 1, kv_len, &L)) return SB_ERR_INVALID_ARG;
  if (ws_bytes < L.total) return SB_ERR_CAPACITY;
  const int c = chain;
  const int R = 1 + c + k_max * depth;
  if ((int64_t)kv_len + R > kv->capacity) return SB_ERR_CAPACITY;
  const int V = draft->cfg.vocab;
  char *ws = (char *)d_ws;
  float *logits = (float *)(ws + L.logits);
  sb_row_stats *stats = (sb_row_stats *)(ws + L.stats);
  int32_t *count = (int32_t *)(ws + L.ints) + 1;
  const size_t fws = L.logits;
  int32_t par[SB_MAX_ROWS];
  par[0] = -1;
  for (int t = 1; t <= c; ++t) par[t] = t - 1;
  // the branch-point candidates into rows c + 1 .. c + B
  sb_status st = sb_branch_candidates(d_q, V, d_xb, k_max, mode, d_u, count, d_tokens + c + 1,
                                      d_q + (size_t)(c + 1) * V, ws + L.branch,
                                      sb_branch_workspace_bytes(), stream);
  if (st != SB_OK) return st;
  int32_t B = 0;
  if (hipMemcpyAsync(&B, count, sizeof(B), hipMemcpyDeviceToHost, stream) != hipSuccess ||
      hipStreamSynchronize(stream) != hipSuccess)
    return SB_ERR_HIP;
  if (B < 0 || B > k_max) return SB_ERR_HIP;
  for (int i = 0; i < B; ++i) par[c + 1 + i] = c;
  // continuations, one depth per step
  int32_t src[SB_BRANCH_MAX_K], dst[SB_BRANCH_MAX_K];
  for (int d = 2; d <= depth && B > 0; ++d) {
    const int n = 1 + c + (d - 1) * B;
    st = sb_verify_forward(draft, kv, kv_len, d_tokens, par, n, temperature, logits, stats, ws, fws,
                           stream);
    if (st != SB_OK) return st;
    for (int i = 0; i < B; ++i) {
      src[i] = c + 1 + (d - 2) * B + i;
      dst[i] = c + 1 + (d - 1) * B + i;
      par[dst[i]] = src[i];
    }
    st = draft_sample_rows(draft, ws, L, temperature, n, B, src, dst, R, d_u + k_max * (d - 1),
                           d_tokens, d_q, nullptr, stream);
    if (st != SB_OK) return st;
  }
  const int n_rows = 1 + c + B * depth;
  for (int i = 0; i < n_rows; ++i) h_parents[i] = par[i];
  *h_branches = B;
  return SB_OK;
}

sb_status sb_draft_round(sb_model *draft, const sb_kv_cache *kv, int32_t kv_len, int32_t k_max,
                         int32_t mode, int32_t depth, int32_t trunk_max, float confidence,
                         float temperature, const float *d_u, int32_t *d_tokens, float *d_q,
                         int32_t *h_parents, int32_t *h_branches, int32_t *h_chain, void *d_ws,
                         size_t ws_bytes, hipStream_t stream) {
  if (!draft_args_ok(draft, kv, temperature) || !d_u || !d_tokens || !d_q || !h_parents ||
      !h_branches || !h_chain || !d_ws || isnan(confidence))
    return SB_ERR_INVALID_ARG;
  if (mode != SB_BRANCH_TOPK && mode != SB_BRANCH_IID && mode != SB_BRANCH_WOR)
    return SB_ERR_INVALID_ARG;
  RoundLayout L;
  if (!round_layout(draft, k_max, depth, trunk_max, kv_len, &L)) return SB_ERR_INVALID_ARG;
  if (ws_bytes < L.total) return SB_ERR_CAPACITY;
  if ((int64_t)kv_len + trunk_max + k_max * depth > kv->capacity) return SB_ERR_CAPACITY;
  // x_b lives in the workspace between the two phases, in the last int of
  // this layout: the two phases lay out smaller rounds (trunk_max rows,
  // then c + 1 <= trunk_max), whose areas end below it, or at its first
  // three ints when the sizes coincide
  int32_t *xb = (int32_t *)((char *)d_ws + L.ints) + 3;
  int32_t c = 0;
  sb_status st = sb_draft_chain(draft, kv, kv_len, trunk_max, confidence, 0, temperature, d_u,
                                d_tokens, d_q, xb, &c, d_ws, ws_bytes, stream);
  if (st != SB_OK) return st;
  st = sb_draft_branches(draft, kv, kv_len, c, xb, k_max, mode, depth, temperature,
                         d_u + trunk_max, d_tokens, d_q, h_parents, h_branches, d_ws, ws_bytes,
                         stream);
  if (st != SB_OK) return st;
  *h_chain = c;
  return SB_OK;
}

sb_status sb_round_finish(int32_t chain, int32_t branches, int32_t depth,
                          const sb_step_result *d_walk, const int32_t *d_select,
                          sb_round_result *d_round, sb_step_result *d_draft_path,
                          hipStream_t stream) {
  if (!d_walk || !d_round || !d_draft_path || chain < 0 || branches < 0 || depth < 1)
    return SB_ERR_INVALID_ARG;
  if (branches > 0 && !d_select) return SB_ERR_INVALID_ARG;
  if ((int64_t)1 + chain + (int64_t)branches * depth > SB_MAX_ROWS) return SB_ERR_INVALID_ARG;
  return hip_status(launch_round_finish(chain, branches, depth, d_walk,
                                        branches > 0 ? d_select : nullptr, d_round, d_draft_path,
                                        stream));
}

// Workspace of a whole round: the draft's round area (its forward, logits,
// statistics, candidates, sampler and x_b), the target's chain forward, the
// target's sampler and the draft's kept-row path.
struct SpecLayout {
  RoundLayout draft;
  size_t target, sample, dpath, total;
};
static bool spec_layout(const sb_model *target, const sb_model *draft, const sb_round_params *p,
                        int t_len, int d_len, SpecLayout *o) {
  if (!target || !draft || !p || target->cfg.vocab != draft->cfg.vocab || t_len < 0) return false;
  if (!round_layout(draft, p->k_max, p->depth, p->trunk_max, d_len, &o->draft)) return false;
  const size_t tw = sb_workspace_bytes(target, p->trunk_max, t_len);
  const size_t sw = sb_sample_workspace_bytes(target->cfg.vocab);
  if (!tw || !sw) return false;
  o->target = align_up(o->draft.total);
  o->sample = o->target + align_up(tw);
  o->dpath = o->sample + align_up(sw);
  o->total = o->dpath + align_up(sizeof(sb_step_result));
  return true;
}

size_t sb_spec_round_workspace_bytes(const sb_model *target, const sb_model *draft,
                                     const sb_round_params *p, int32_t t_len, int32_t d_len) {
  SpecLayout L;
  return spec_layout(target, draft, p, t_len, d_len, &L) ? L.total : 0;
}

namespace {
// An event that is destroyed with its scope (the work it marks may still
// be pending; HIP releases it once that work completes).
struct ScopedEvent {
  hipEvent_t e = nullptr;
  hipError_t make() { return hipEventCreateWithFlags(&e, hipEventDisableTiming); }
  ~ScopedEvent() {
    if (e) (void)hipEventDestroy(e);
  }
};
}  // namespace

sb_status sb_spec_round(sb_model *target, const sb_kv_cache *t_kv, int32_t t_len, sb_model *draft,
                        const sb_kv_cache *d_kv, int32_t d_len, const sb_round_params *p,
                        const float *d_u_draft, const float *d_u_walk, const float *d_u_sel,
                        int32_t *d_tokens, float *d_q, float *d_logits, sb_row_stats *d_stats,
                        sb_step_result *d_walk, int32_t *d_select, sb_round_result *d_round,
                        int32_t *d_new_lens, int32_t *h_parents, int32_t *h_chain,
                        int32_t *h_branches, void *d_ws, size_t ws_bytes,
                        hipStream_t verify_stream, hipStream_t draft_stream) {
  if (!target || !draft || target == draft || !t_kv || !d_kv || !p || !d_u_draft || !d_u_walk ||
      !d_u_sel || !d_tokens || !d_q || !d_logits || !d_stats || !d_walk || !d_select ||
      !d_round || !d_new_lens || !h_parents || !h_chain || !h_branches || !d_ws)
    return SB_ERR_INVALID_ARG;
  if (!t_kv->k || !t_kv->v || !temperature_ok(p->temperature) || isnan(p->confidence) ||
      (p->flags & ~SB_CHAIN_CONDITIONED) != 0)
    return SB_ERR_INVALID_ARG;
  SpecLayout L;
  if (!spec_layout(target, draft, p, t_len, d_len, &L)) return SB_ERR_INVALID_ARG;
  if (ws_bytes < L.total) return SB_ERR_CAPACITY;
  if ((int64_t)t_len + p->trunk_max > t_kv->capacity) return SB_ERR_CAPACITY;
  const int V = target->cfg.vocab;
  const float T = p->temperature;
  char *ws = (char *)d_ws;
  int32_t *xb = (int32_t *)(ws + L.draft.ints) + 3;  // as sb_draft_round keeps it
  sb_step_result *dpath = (sb_step_result *)(ws + L.dpath);
  ScopedEvent chain_done, branches_done;
  if (chain_done.make() != hipSuccess || branches_done.make() != hipSuccess) return SB_ERR_HIP;

  // drafting phase: the chain up to the branch point
  int32_t c = 0;
  sb_status st = sb_draft_chain(draft, d_kv, d_len, p->trunk_max, p->confidence, p->flags, T,
                                d_u_draft, d_tokens, d_q, xb, &c, ws, L.draft.total, draft_stream);
  if (st != SB_OK) return st;
  if (hipEventRecord(chain_done.e, draft_stream) != hipSuccess ||
      hipStreamWaitEvent(verify_stream, chain_done.e, 0) != hipSuccess)
    return SB_ERR_HIP;

  // verification phase: the target scores and tests the chain ...
  int32_t par[SB_MAX_ROWS];
  par[0] = -1;
  for (int t = 1; t <= c; ++t) par[t] = t - 1;
  st = sb_verify_forward(target, t_kv, t_len, d_tokens, par, c + 1, T, d_logits, d_stats,
                         ws + L.target, L.sample - L.target, verify_stream);
  if (st != SB_OK) return st;
  st = sb_accept_resample(V, c + 1, d_tokens, par, d_logits, d_stats, T, d_q, d_u_walk, d_walk,
                          ws + L.sample, L.dpath - L.sample, verify_stream);
  if (st != SB_OK) return st;
  // ... while the draft branches at x_b on its own stream
  int32_t B = 0;
  st = sb_draft_branches(draft, d_kv, d_len, c, xb, p->k_max, p->mode, p->depth, T,
                         d_u_draft + p->trunk_max, d_tokens, d_q, h_parents, &B, ws,
                         L.draft.total, draft_stream);
  if (st != SB_OK) return st;
  if (hipEventRecord(branches_done.e, draft_stream) != hipSuccess ||
      hipStreamWaitEvent(verify_stream, branches_done.e, 0) != hipSuccess)
    return SB_ERR_HIP;

  // Algorithm 1 at the chain's last row, then both rollbacks
  if (B > 0) {
    st = sb_select_branch(V, d_logits + (size_t)c * V, d_stats + c, T, B, d_tokens + c + 1,
                          d_q + (size_t)(c + 1) * V, d_u_sel, d_select, ws + L.sample,
                          L.dpath - L.sample, verify_stream);
    if (st != SB_OK) return st;
  }
  st = sb_round_finish(c, B, p->depth, d_walk, B > 0 ? d_select : nullptr, d_round, dpath,
                       verify_stream);
  if (st != SB_OK) return st;
  st = sb_kv_rollback(target, t_kv, t_len, d_walk, d_new_lens, verify_stream);
  if (st != SB_OK) return st;
  st = sb_kv_rollback(draft, d_kv, d_len, dpath, d_new_lens + 1, verify_stream);
  if (st != SB_OK) return st;
  *h_chain = c;
  *h_branches = B;
  return SB_OK;
}

sb_status sb_kv_rollback(const sb_model *m, const sb_kv_cache *kv, int32_t kv_len,
                         const sb_step_result *d_result, int32_t *d_new_len,
                         hipStream_t stream) {
  if (!m || !kv || !kv->k || !kv->v || !d_result || !d_new_len) return SB_ERR_INVALID_ARG;
  if (kv_len < 0 || kv_len >= kv->capacity) return SB_ERR_CAPACITY;
  if (kv->capacity % 8 != 0) return SB_ERR_CAPACITY;
  const sb_model_config &c = m->cfg;
  return hip_status(launch_rollback(c.n_layers, c.n_kv_heads, kv->capacity, c.head_dim,
                                    (int)elem_bytes(c), kv->k, kv->v, kv_len, d_result, d_new_len,
                                    stream));
}

}  // extern "C"
