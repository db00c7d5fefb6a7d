// Launch planning and dispatch of the skinny matrix-core GEMM (the kernel
// is in sb_gemm_kernel.h, built once per epilogue kind in k_gemm_*.hip).
//
// The residual projections, about one tile per compute unit, split K across
// workgroups and leave partial deltas for the next RMSNorm (RESID), or run
// unsplit and apply the following RMSNorm themselves (RESID_NORM).
#include "sb_internal_fwd.h"

namespace sb {

namespace {

int device_cus() {
  static int cus = 0;
  if (cus == 0) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        cus <= 0)
      cus = 256;
  }
  return cus;
}

// Token-tile counts and tiles per pass with a kernel (token tiles rounded
// up; padded rows read as zero).  A kernel for 5 token tiles (65 .. 80
// rows) took the 13B step at 65 rows and prefix 8192 from 9.36 to 9.24 ms
// against padding to 6.
constexpr int kTTs[] = {1, 2, 3, 4, 5, 6, 8, 12, 16};
constexpr int kNTs[] = {1, 2, 3, 4, 6, 8};

}  // namespace

// Token tiles past which the projections take k_gemm_wide (from 5 token
// tiles, 13B at 65 rows: QKV 35 -> 46 us, down 37 -> 41, gate/up 61 -> 61).
constexpr int kWideFrom = 8;

GemmPlan plan_gemm(int epi, int tiles, int ks, int n_tok) {
  GemmPlan p{};
  const int nc = ks / 8;
  const int tt_all = (n_tok + 15) / 16;
  // Wide trees: k_gemm_wide (a wave owns a tile pair over one of KS parts
  // of the workgroup's K range; the activation is staged once per 16 / KS
  // tiles through LDS).  QKV and the residual projections, with the fewest
  // tiles, take KS = 4; the residual projections also split K over up to
  // kMaxSplit workgroups per tile group.  The LM head runs without its
  // fused statistics (the separate pass reads the logits).  13B at 129
  // rows: gate/up 120 -> 78 us, QKV 69 -> 61, down 61 -> 50 (KS = 2; KS = 4
  // took the step from 13.20 to 13.11 ms), the LM head 138 + 5 -> 79 + 11
  // with the statistics pass.
  if (tt_all > kWideFrom &&
      (epi == EPI_QKV || epi == EPI_SWIGLU || epi == EPI_RESID || epi == EPI_LOGITS)) {
    const int KS = (epi == EPI_QKV || epi == EPI_RESID) ? 4 : 2;
    p.wide = KS;
    p.tt = tt_all <= 9 ? 9 : tt_all <= 12 ? 12 : 16;
    p.nt = 2;
    p.groups = (tiles + 16 / KS - 1) / (16 / KS);
    int S = 1;
    if (epi == EPI_RESID) {
      S = device_cus() / p.groups;
      if (S > kMaxSplit) S = kMaxSplit;
      if (S * KS > ks) S = ks / KS;
      if (S < 1) S = 1;
    }
    p.split = S;
    p.grid = p.groups * S;
    return p;
  }
  const int cus = device_cus();
  for (int v : kTTs)
    if (v >= tt_all) {
      p.tt = v;
      break;
    }
  // Projections that add into the residual stream have as many tiles as the
  // model is wide, about one per compute unit: they split K so that each
  // workgroup owns several tiles; the next RMSNorm sums the partial deltas.
  const int per_cu = (tiles + cus - 1) / cus;
  int S = 1;
  if (epi == EPI_RESID) S = per_cu == 1 ? kMaxSplit : per_cu == 2 ? 2 : 1;  // RESID_NORM: 1
  if (S > nc) S = nc;
  if (S < 1) S = 1;
  int groups = cus / S;
  if (groups > tiles) groups = tiles;
  const int per_wg = (tiles + groups - 1) / groups;
  const int cap = gemm_nt_cap(p.tt);
  const int passes = (per_wg + cap - 1) / cap;
  const int need = (per_wg + passes - 1) / passes;
  for (int v : kNTs)
    if (v >= need) {
      p.nt = v;
      break;
    }
  p.split = S;
  p.groups = groups;
  p.grid = groups * S;
  return p;
}

bool resid_norm_fusable(int tiles, int ks, int n_tok, int *groups) {
  const GemmPlan p = plan_gemm(EPI_RESID_NORM, tiles, ks, n_tok);
  if (groups) *groups = p.groups;
  return n_tok <= kNormFuseRows && p.groups <= kSsGroups &&
         (tiles + p.groups - 1) / p.groups <= p.nt && p.nt * p.tt <= kRedPairs;
}

hipError_t launch_gemm(int epi, const GemmArgs &a, int tiles, int *split, hipStream_t s) {
  if (a.ks % 8 != 0 || a.n_tok <= 0 || a.n_tok > SB_MAX_ROWS) return hipErrorInvalidValue;
  if (epi == EPI_RESID_NORM && (!resid_norm_fusable(tiles, a.ks, a.n_tok, nullptr) || !a.gain ||
                                !a.xn || !a.ss || a.xn_ks * 32 < a.out_rows))
    return hipErrorInvalidValue;
  if (a.ss_in && (a.n_tok > kNormFuseRows || a.ss_groups < 1 || a.ss_groups > kSsGroups ||
                  epi == EPI_RESID_NORM || epi == EPI_QKV))
    return hipErrorInvalidValue;
  const GemmPlan p = plan_gemm(epi, tiles, a.ks, a.n_tok);
  // k_gemm_wide has no fused softmax statistics: the caller runs the
  // separate pass for such shapes
  if (p.wide && a.lm_part) return hipErrorInvalidValue;
  GemmArgs b = a;
  b.epi = epi;
  b.tiles = tiles;
  b.split = p.split;
  b.groups = p.groups;
  if (split) *split = p.split;
  switch (epi) {
    case EPI_QKV: return launch_gemm_qkv(b, p, s);
    case EPI_RESID: return launch_gemm_resid(b, p, s);
    case EPI_SWIGLU: return launch_gemm_swiglu(b, p, s);
    case EPI_LOGITS: return launch_gemm_logits(b, p, s);
    case EPI_RESID_NORM: return launch_gemm_resid_norm(b, p, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace sb
