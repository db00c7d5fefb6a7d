// Branch-point candidates (Section "Branch Resampling"): at an unconfident
// draft token x_b the draft side spawns B = max(1, floor(k_max (1 - q(x_b))))
// sibling first tokens from the draft distribution q at that position, capped
// by the number of tokens with q > 0.  Each candidate carries the distribution
// it was drawn from, since verification (Algorithm 1) subtracts exactly that
// from p:
//   top-k  the B largest entries (lowest index first on ties), one-hot rows;
//   i.i.d. B inverse-CDF draws from q, each carrying q;
//   w/o replacement  draw i from q with the earlier candidates zeroed,
//          carrying that remainder divided by its float64 mass.
//
// One workgroup (k_branch_select) builds a two-level summary of q in LDS
// (and keeps q itself there when it fits):
// level 1 holds, per chunk of 256 tokens, the float64 sum (draws) or the
// maximum (top-k) of the chunk; level 2 the same over 64 level-1 entries.  A
// draw or a top-k pick is then one wave descending the summary: 64 level-2
// entries, 64 level-1 entries, 64 lanes of 4 tokens, each level a 64-lane
// scan (or maximum) and a ballot.  Removing a candidate recomputes its chunk
// and its level-2 entry from their parts in the order they were built, so the
// summary always equals a fresh build over the remainder.  A second, wide
// kernel (k_branch_rows) writes the B carried rows.
#include <climits>

#include "sb_device.h"
#include "sb_internal_fwd.h"

namespace sb {
namespace {

constexpr int kSelThreads = 1024;
constexpr int kSelWaves = kSelThreads / 64;
constexpr int kChunk = 256;                 // tokens per level-1 entry (4 per lane)
constexpr int kMaxL1 = 64 * 64;             // level-1 entries (64 per level-2 entry)
constexpr int kBuildUnroll = 8;             // chunks in flight per wave while building
constexpr int kRowThreads = 256;
static_assert(SB_BRANCH_MAX_K <= kSelWaves, "one wave per i.i.d. draw");
static_assert((long)kMaxL1 * kChunk >= SB_BRANCH_MAX_VOCAB, "summary covers the vocabulary");

// ---- wave collectives on DPP -------------------------------------------
// A float64 moves as two 32-bit DPP lanes.  Lanes whose DPP source is
// outside their row of 16 read 0.
template <int kCtrl>
__device__ __forceinline__ double dpp_d(double v) {
  const uint64_t b = __builtin_bit_cast(uint64_t, v);
  const uint32_t lo = (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)b, kCtrl, 0xf, 0xf, false);
  const uint32_t hi =
      (uint32_t)__builtin_amdgcn_update_dpp(0, (int)(uint32_t)(b >> 32), kCtrl, 0xf, 0xf, false);
  return __builtin_bit_cast(double, ((uint64_t)hi << 32) | lo);
}
__device__ __forceinline__ double readlane_d(double v, int l) {
  const uint64_t b = __builtin_bit_cast(uint64_t, v);
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)b, l);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(b >> 32), l);
  return __builtin_bit_cast(double, ((uint64_t)hi << 32) | lo);
}
constexpr int kDppQuadXor1 = 0xB1;     // quad_perm [1,0,3,2]
constexpr int kDppQuadXor2 = 0x4E;     // quad_perm [2,3,0,1]
constexpr int kDppRowHalfMirror = 0x141;
constexpr int kDppRowMirror = 0x140;
constexpr int kDppRowShr = 0x110;      // + shift

// Sum (or maximum) over the wave: pairs within quads, then the two quads of
// each half-row, then the two halves of each row (every pairing adds the
// same two values in either order, so all lanes of a row hold the same
// total), then the four row totals in row order.  Every lane returns the
// same value, and the same lane values always give the same result.
template <bool kMax>
__device__ __forceinline__ double wave_red_d(double v) {
  auto op = [](double a, double b) { return kMax ? fmax(a, b) : a + b; };
  v = op(v, dpp_d<kDppQuadXor1>(v));
  v = op(v, dpp_d<kDppQuadXor2>(v));
  v = op(v, dpp_d<kDppRowHalfMirror>(v));
  v = op(v, dpp_d<kDppRowMirror>(v));
  return op(op(op(readlane_d(v, 0), readlane_d(v, 16)), readlane_d(v, 32)), readlane_d(v, 48));
}
__device__ __forceinline__ double wave_sum_d(double v) { return wave_red_d<false>(v); }
__device__ __forceinline__ double wave_max_d(double v) { return wave_red_d<true>(v); }

// Inclusive scan over the wave: shifts of 1, 2, 4, 8 within each row, then
// the totals of the rows ahead.
__device__ __forceinline__ double wave_scan_d(double x) {
  x += dpp_d<kDppRowShr + 1>(x);
  x += dpp_d<kDppRowShr + 2>(x);
  x += dpp_d<kDppRowShr + 4>(x);
  x += dpp_d<kDppRowShr + 8>(x);
  const double t0 = readlane_d(x, 15), t1 = readlane_d(x, 31), t2 = readlane_d(x, 47);
  const int row = (threadIdx.x & 63) >> 4;
  const double t01 = t0 + t1;
  return row == 0 ? x : x + (row == 1 ? t0 : row == 2 ? t01 : t01 + t2);
}

// Among lanes with a > 0, the first whose inclusive prefix exceeds thr; when
// rounding leaves none, the last lane with a > 0 (0 if no lane has mass, which
// a parent with mass rules out).  *before is the prefix ahead of that lane.
__device__ __forceinline__ int pick_sum(double a, double thr, double *before) {
  const double inc = wave_scan_d(a);
  const unsigned long long hit = __ballot(a > 0.0 && inc > thr);
  int sel;
  if (hit) {
    sel = __ffsll((long long)hit) - 1;
  } else {
    const unsigned long long pos = __ballot(a > 0.0);
    sel = pos ? 63 - __clzll((long long)pos) : 0;
  }
  *before = readlane_d(inc - a, sel);
  return sel;
}

// The lowest lane holding the wave's maximum of a.
__device__ __forceinline__ int pick_max(double a) {
  const double m = wave_max_d(a);
  return __ffsll((long long)__ballot(a == m)) - 1;
}

// kLds: the vocabulary fits in LDS (at most kLdsVocab tokens) and q is kept
// there after the first pass, so a pick reads no global memory.
constexpr int kLdsVocab = 32768;
template <bool kLds>
struct SelShared {
  double s1[kLds ? kLdsVocab / kChunk : kMaxL1];
  double s2[64];
  int cnt[kSelWaves];
  __attribute__((aligned(16))) float qs[kLds ? kLdsVocab : 4];
};

// The 4 tokens of lane `lane` in chunk c: q where it counts, else the empty
// value (0 for sums, -1 for top-k keys).  Taken candidates count as empty.
// From global memory (and kept in LDS when kLds) or, with from_lds, from LDS.
template <bool kLds>
__device__ __forceinline__ void chunk_vals(const BranchArgs &a, __amdgpu_buffer_rsrc_t qrs,
                                           SelShared<kLds> &sh, int c, int lane, bool from_lds,
                                           int my_taken, int n_taken, double (&x)[4]) {
  const int v0 = c * kChunk + lane * 4;
  float f[4];
  if (kLds && from_lds) {
    const f32x4 t = *(const f32x4 *)&sh.qs[v0 < a.vocab ? v0 : 0];
#pragma unroll
    for (int j = 0; j < 4; ++j) f[j] = t[j];
  } else if (a.vec4) {
    const f32x4 t = __builtin_bit_cast(
        f32x4, __builtin_amdgcn_raw_buffer_load_b128(qrs, v0 < a.vocab ? v0 * 4 : a.vocab * 4, 0, 0));
#pragma unroll
    for (int j = 0; j < 4; ++j) f[j] = t[j];
  } else {
#pragma unroll
    for (int j = 0; j < 4; ++j)
      f[j] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(
                                           qrs, v0 + j < a.vocab ? (v0 + j) * 4 : a.vocab * 4, 0, 0));
  }
  if (kLds && !from_lds && v0 < kLdsVocab) *(f32x4 *)&sh.qs[v0] = f32x4{f[0], f[1], f[2], f[3]};
  const double empty = a.mode == SB_BRANCH_TOPK ? -1.0 : 0.0;
  bool in[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) in[j] = v0 + j < a.vocab;
  // the taken candidates that fall in this chunk (lane i holds candidate i)
  unsigned long long hits = __ballot(lane < n_taken && my_taken / kChunk == c);
  while (hits) {
    const int i = __ffsll((long long)hits) - 1;
    hits &= hits - 1;
    const int t = __builtin_amdgcn_readlane(my_taken, i);
#pragma unroll
    for (int j = 0; j < 4; ++j) in[j] = in[j] && v0 + j != t;
  }
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    if (a.mode == SB_BRANCH_TOPK)
      x[j] = in[j] ? (double)f[j] : empty;
    else
      x[j] = in[j] && f[j] > 0.0f ? (double)f[j] : 0.0;
  }
}

__device__ __forceinline__ double lane_key(const BranchArgs &a, const double (&x)[4]) {
  if (a.mode == SB_BRANCH_TOPK) return fmax(fmax(x[0], x[1]), fmax(x[2], x[3]));
  return ((x[0] + x[1]) + x[2]) + x[3];
}

// Level entry reads: the empty value beyond the last entry.
__device__ __forceinline__ double level_val(const BranchArgs &a, const double *s, int idx, int n) {
  return idx < n ? s[idx] : (a.mode == SB_BRANCH_TOPK ? -1.0 : 0.0);
}

// The token within lane e's 4 (x as that lane holds them): the first whose
// running sum exceeds thr, else the lane's last token with mass.
__device__ __forceinline__ int lane_draw(const double (&x)[4], double thr, int e) {
  int pick = -1, last = -1;
  double run = 0.0;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    run += x[j];
    if (x[j] > 0.0) {
      last = j;
      if (pick < 0 && run > thr) pick = j;
    }
  }
  return __builtin_amdgcn_readlane(pick >= 0 ? pick : max(last, 0), e);
}

template <bool kLds>
__global__ __launch_bounds__(kSelThreads) void k_branch_select(BranchArgs a) {
  __shared__ SelShared<kLds> sh;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int n1 = (a.vocab + kChunk - 1) / kChunk;
  const int n2 = (n1 + 63) / 64;
  const __amdgpu_buffer_rsrc_t qrs = uniform_rsrc(a.q, a.vocab * 4);
  // q(x_b), fetched first so its latency hides under the first pass
  const int xb = *a.x_b;
  const float qxb = __builtin_bit_cast(
      float, __builtin_amdgcn_raw_buffer_load_b32(qrs, xb >= 0 && xb < a.vocab ? xb * 4 : a.vocab * 4,
                                                  0, 0));

  // level 1 (and the count of tokens with mass), kBuildUnroll chunks per wave in flight
  int cnt = 0;
  for (int c0 = w; c0 < n1; c0 += kSelWaves * kBuildUnroll) {
    double x[kBuildUnroll][4];
#pragma unroll
    for (int u = 0; u < kBuildUnroll; ++u) {
      const int c = c0 + u * kSelWaves;
      chunk_vals<kLds>(a, qrs, sh, c < n1 ? c : n1, lane, false, -1, 0, x[u]);
    }
#pragma unroll
    for (int u = 0; u < kBuildUnroll; ++u) {
      const int c = c0 + u * kSelWaves;
      if (c < n1) {
        for (int j = 0; j < 4; ++j) cnt += x[u][j] > 0.0;
        const double k1 = a.mode == SB_BRANCH_TOPK ? wave_max_d(lane_key(a, x[u]))
                                                   : wave_sum_d(lane_key(a, x[u]));
        if (lane == 0) sh.s1[c] = k1;
      }
    }
  }
  for (int o = 32; o > 0; o >>= 1) cnt += __shfl_xor(cnt, o, 64);
  if (lane == 0) sh.cnt[w] = cnt;
  __syncthreads();
  // level 2
  for (int j = w; j < n2; j += kSelWaves) {
    const double v = level_val(a, sh.s1, j * 64 + lane, n1);
    const double k2 = a.mode == SB_BRANCH_TOPK ? wave_max_d(v) : wave_sum_d(v);
    if (lane == 0) sh.s2[j] = k2;
  }
  __syncthreads();

  // B = max(1, floor(k_max (1 - q(x_b)))), at most the tokens with mass and k_max
  int nnz = 0;
  for (int i = 0; i < kSelWaves; ++i) nnz += sh.cnt[i];
  const double bf = floor((double)a.k_max * (1.0 - (double)qxb));
  int B = bf >= 1.0 ? (bf <= (double)a.k_max ? (int)bf : a.k_max) : 1;
  B = min(B, nnz);

  if (a.mode == SB_BRANCH_IID) {
    // independent draws from q: wave i takes draw i
    if (w < B) {
      const double a2 = level_val(a, sh.s2, lane, n2);
      const double W = wave_sum_d(a2);
      double thr = (double)a.u[w] * W, before;
      const int c2 = pick_sum(a2, thr, &before);
      thr -= before;
      const int c1 = c2 * 64 + pick_sum(level_val(a, sh.s1, c2 * 64 + lane, n1), thr, &before);
      thr -= before;
      double x[4];
      chunk_vals<kLds>(a, qrs, sh, c1, lane, true, -1, 0, x);
      const int e = pick_sum(lane_key(a, x), thr, &before);
      thr -= before;
      const int jj = lane_draw(x, thr, e);
      if (lane == 0) a.tokens[w] = c1 * kChunk + e * 4 + jj;
    }
  } else if (w == 0) {
    // top-k picks or draws without replacement, one after another on wave 0
    int my_taken = -1;
    for (int i = 0; i < B; ++i) {
      const double a2 = level_val(a, sh.s2, lane, n2);
      double thr = 0.0, before = 0.0;
      int c2;
      if (a.mode == SB_BRANCH_TOPK) {
        c2 = pick_max(a2);
      } else {
        const double Z = wave_sum_d(a2);
        if (lane == 0) a.znorm[i] = Z;
        thr = (double)a.u[i] * Z;
        c2 = pick_sum(a2, thr, &before);
        thr -= before;
      }
      const double a1 = level_val(a, sh.s1, c2 * 64 + lane, n1);
      int l1;
      if (a.mode == SB_BRANCH_TOPK) {
        l1 = pick_max(a1);
      } else {
        l1 = pick_sum(a1, thr, &before);
        thr -= before;
      }
      const int c1 = c2 * 64 + l1;
      double x[4];
      chunk_vals<kLds>(a, qrs, sh, c1, lane, true, my_taken, i, x);
      const double k0 = lane_key(a, x);
      int e, jj;
      if (a.mode == SB_BRANCH_TOPK) {
        e = pick_max(k0);
        int f = 0;
        for (int j = 3; j >= 0; --j)
          if (x[j] == k0) f = j;
        jj = __builtin_amdgcn_readlane(f, e);
      } else {
        e = pick_sum(k0, thr, &before);
        thr -= before;
        jj = lane_draw(x, thr, e);
      }
      const int tok = c1 * kChunk + e * 4 + jj;
      // take it out of the summary: its chunk, then its level-2 entry, each
      // rebuilt from its parts as the first build did
      if (lane == e) {
#pragma unroll
        for (int j = 0; j < 4; ++j)
          if (j == jj) x[j] = a.mode == SB_BRANCH_TOPK ? -1.0 : 0.0;
      }
      const double n1v = a.mode == SB_BRANCH_TOPK ? wave_max_d(lane_key(a, x))
                                                  : wave_sum_d(lane_key(a, x));
      const double a1n = lane == l1 ? n1v : a1;
      const double n2v = a.mode == SB_BRANCH_TOPK ? wave_max_d(a1n) : wave_sum_d(a1n);
      if (lane == i) my_taken = tok;
      if (lane == 0) {
        sh.s1[c1] = n1v;
        sh.s2[c2] = n2v;
        a.tokens[i] = tok;
      }
      __builtin_amdgcn_wave_barrier();  // one wave's LDS writes land before its next reads
    }
  }
  if (threadIdx.x == 0) *a.count = B;
  for (int i = B + (int)threadIdx.x; i < a.k_max; i += kSelThreads) a.tokens[i] = -1;
}

// Row i of the carried distributions, 8 tokens per thread (two float4 when
// the row is 16-byte aligned).
__global__ __launch_bounds__(kRowThreads) void k_branch_rows(BranchArgs a) {
  __shared__ int toks[SB_BRANCH_MAX_K];
  const int i = blockIdx.y;
  // the count, the candidates, Z and this thread's q are loaded together (all
  // in bounds whatever the count is); the count then decides
  const int B = *a.count;
  if ((int)threadIdx.x < a.k_max) toks[threadIdx.x] = a.tokens[threadIdx.x];
  const double Z = a.mode == SB_BRANCH_WOR ? a.znorm[i] : 1.0;
  const int base = blockIdx.x * kRowThreads * 8;
  float qv[8];
  if (a.vec4) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int v0 = base + (h * kRowThreads + (int)threadIdx.x) * 4;
      const f32x4 t = v0 < a.vocab ? *(const f32x4 *)(a.q + v0) : f32x4{0, 0, 0, 0};
#pragma unroll
      for (int j = 0; j < 4; ++j) qv[4 * h + j] = t[j];
    }
  } else {
#pragma unroll
    for (int h = 0; h < 8; ++h) {
      const int v = base + h * kRowThreads + (int)threadIdx.x;
      qv[h] = v < a.vocab ? a.q[v] : 0.0f;
    }
  }
  __syncthreads();
  if (i >= B) return;
  float *row = a.rows + (size_t)i * a.vocab;
  auto value = [&](int v, float q) -> float {
    if (a.mode == SB_BRANCH_TOPK) return v == toks[i] ? 1.0f : 0.0f;
    if (a.mode == SB_BRANCH_IID) return q;
    for (int j = 0; j < i; ++j)
      if (v == toks[j]) return 0.0f;
    return (float)((double)q / Z);
  };
  if (a.vec4) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int v0 = base + (h * kRowThreads + (int)threadIdx.x) * 4;
      if (v0 < a.vocab) {
        f32x4 o;
#pragma unroll
        for (int j = 0; j < 4; ++j) o[j] = value(v0 + j, qv[4 * h + j]);
        *(f32x4 *)(row + v0) = o;
      }
    }
  } else {
#pragma unroll
    for (int h = 0; h < 8; ++h) {
      const int v = base + h * kRowThreads + (int)threadIdx.x;
      if (v < a.vocab) row[v] = value(v, qv[h]);
    }
  }
}

}  // namespace

hipError_t launch_branch(const BranchArgs &a, hipStream_t s) {
  if (a.vocab <= kLdsVocab)
    hipLaunchKernelGGL(k_branch_select<true>, dim3(1), dim3(kSelThreads), 0, s, a);
  else
    hipLaunchKernelGGL(k_branch_select<false>, dim3(1), dim3(kSelThreads), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int cols = (a.vocab + kRowThreads * 8 - 1) / (kRowThreads * 8);
  hipLaunchKernelGGL(k_branch_rows, dim3(cols, a.k_max), dim3(kRowThreads), 0, s, a);
  return hipGetLastError();
}

}  // namespace sb
