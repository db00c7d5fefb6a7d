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
// One workgroup (k_branch_select) builds a two-level summary of q in LDS:
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

// Sum over the wave by an xor butterfly: every lane ends with the same value,
// and the same lane values always give the same sum.
__device__ __forceinline__ double wave_sum_d(double v) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
__device__ __forceinline__ double wave_max_d(double v) {
  for (int o = 32; o > 0; o >>= 1) v = fmax(v, __shfl_xor(v, o, 64));
  return v;
}

// Among lanes with a > 0, the first whose inclusive prefix exceeds thr; when
// rounding leaves none, the last lane with a > 0 (0 if no lane has mass, which
// a parent with mass rules out).  *before is the prefix ahead of that lane.
__device__ __forceinline__ int pick_sum(double a, double thr, double *before) {
  const int lane = threadIdx.x & 63;
  double inc = a;
  for (int o = 1; o < 64; o <<= 1) {
    const double y = __shfl_up(inc, o, 64);
    if (lane >= o) inc += y;
  }
  const unsigned long long hit = __ballot(a > 0.0 && inc > thr);
  int sel;
  if (hit) {
    sel = __ffsll((long long)hit) - 1;
  } else {
    const unsigned long long pos = __ballot(a > 0.0);
    sel = pos ? 63 - __clzll((long long)pos) : 0;
  }
  *before = __shfl(inc - a, sel, 64);
  return sel;
}

// The lowest lane holding the wave's maximum of a.
__device__ __forceinline__ int pick_max(double a) {
  const double m = wave_max_d(a);
  return __ffsll((long long)__ballot(a == m)) - 1;
}

struct SelShared {
  double s1[kMaxL1];
  double s2[64];
  int tok[SB_BRANCH_MAX_K];
  int cnt[kSelWaves];
};

// The 4 tokens of lane `lane` in chunk c: q where it counts, else the empty
// value (0 for sums, -1 for top-k keys).  Taken candidates count as empty.
__device__ __forceinline__ void chunk_vals(const BranchArgs &a, __amdgpu_buffer_rsrc_t qrs, int c,
                                           int lane, const int *taken, int n_taken, double (&x)[4]) {
  const int v0 = c * kChunk + lane * 4;
  float f[4];
  if (a.vec4) {
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
  const double empty = a.mode == SB_BRANCH_TOPK ? -1.0 : 0.0;
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int v = v0 + j;
    bool in = v < a.vocab;
    for (int i = 0; i < n_taken; ++i) in = in && v != taken[i];
    if (a.mode == SB_BRANCH_TOPK)
      x[j] = in ? (double)f[j] : empty;
    else
      x[j] = in && f[j] > 0.0f ? (double)f[j] : 0.0;
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

__global__ __launch_bounds__(kSelThreads) void k_branch_select(BranchArgs a) {
  __shared__ SelShared sh;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int n1 = (a.vocab + kChunk - 1) / kChunk;
  const int n2 = (n1 + 63) / 64;
  const __amdgpu_buffer_rsrc_t qrs = uniform_rsrc(a.q, a.vocab * 4);

  // level 1 (and the count of tokens with mass), kBuildUnroll chunks per wave in flight
  int cnt = 0;
  for (int c0 = w; c0 < n1; c0 += kSelWaves * kBuildUnroll) {
    double x[kBuildUnroll][4];
#pragma unroll
    for (int u = 0; u < kBuildUnroll; ++u) {
      const int c = c0 + u * kSelWaves;
      chunk_vals(a, qrs, c < n1 ? c : n1, lane, nullptr, 0, x[u]);
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
  const int xb = *a.x_b;
  const float qxb = xb >= 0 && xb < a.vocab ? a.q[xb] : 0.0f;
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
      chunk_vals(a, qrs, c1, lane, nullptr, 0, x);
      const int e = pick_sum(lane_key(a, x), thr, &before);
      thr -= before;
      // the token within lane e's 4: first whose running sum exceeds thr,
      // else its last one with mass
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
      const int jj = __shfl(pick >= 0 ? pick : max(last, 0), e, 64);
      if (lane == 0) a.tokens[w] = c1 * kChunk + e * 4 + jj;
    }
  } else if (w == 0) {
    // top-k picks or draws without replacement, one after another on wave 0
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
      chunk_vals(a, qrs, c1, lane, sh.tok, i, x);
      const double k0 = lane_key(a, x);
      int e, jj;
      if (a.mode == SB_BRANCH_TOPK) {
        e = pick_max(k0);
        int f = 0;
        for (int j = 3; j >= 0; --j)
          if (x[j] == k0) f = j;
        jj = __shfl(f, e, 64);
      } else {
        e = pick_sum(k0, thr, &before);
        thr -= before;
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
        jj = __shfl(pick >= 0 ? pick : max(last, 0), e, 64);
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
      if (lane == 0) {
        sh.s1[c1] = n1v;
        sh.s2[c2] = n2v;
        sh.tok[i] = tok;
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
  const int B = *a.count;
  if (i >= B) return;
  if ((int)threadIdx.x <= i) toks[threadIdx.x] = a.tokens[threadIdx.x];
  __syncthreads();
  const double Z = a.mode == SB_BRANCH_WOR ? a.znorm[i] : 1.0;
  float *row = a.rows + (size_t)i * a.vocab;
  auto value = [&](int v, float qv) -> float {
    if (a.mode == SB_BRANCH_TOPK) return v == toks[i] ? 1.0f : 0.0f;
    if (a.mode == SB_BRANCH_IID) return qv;
    for (int j = 0; j < i; ++j)
      if (v == toks[j]) return 0.0f;
    return (float)((double)qv / Z);
  };
  const int base = blockIdx.x * kRowThreads * 8;
  if (a.vec4) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int v0 = base + (h * kRowThreads + (int)threadIdx.x) * 4;
      if (v0 < a.vocab) {
        const f32x4 qv = *(const f32x4 *)(a.q + v0);
        f32x4 o;
#pragma unroll
        for (int j = 0; j < 4; ++j) o[j] = value(v0 + j, qv[j]);
        *(f32x4 *)(row + v0) = o;
      }
    }
  } else {
#pragma unroll
    for (int h = 0; h < 8; ++h) {
      const int v = base + h * kRowThreads + (int)threadIdx.x;
      if (v < a.vocab) row[v] = value(v, a.q[v]);
    }
  }
}

}  // namespace

hipError_t launch_branch(const BranchArgs &a, hipStream_t s) {
  hipLaunchKernelGGL(k_branch_select, dim3(1), dim3(kSelThreads), 0, s, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int cols = (a.vocab + kRowThreads * 8 - 1) / (kRowThreads * 8);
  hipLaunchKernelGGL(k_branch_rows, dim3(cols, a.k_max), dim3(kRowThreads), 0, s, a);
  return hipGetLastError();
}

}  // namespace sb
