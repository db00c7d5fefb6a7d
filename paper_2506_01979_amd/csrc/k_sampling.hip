// Row softmax statistics, Branch Speculative Sampling at one node, and the
// accept/resample walk over a token tree.
//
// What is computed (Preliminaries, "Speculative Decoding"; Appendix,
// Algorithm 1 "Branch Speculative Sampling"):
//   p(v)   = fl32(exp(fl32(fl32(l_v * fl32(1/T)) - zmax))) / total  (float64)
//            or the one-hot at argmax when T = 0;
//   accept = float64(u) < p~(x) / float64(q(x));
//   reject : p~ <- max(0, p~ - q) / Z,  Z = sum max(0, p~ - q)   (float64),
//            Z <= 0 keeps p~ and raises SB_FLAG_ZERO_RESIDUAL;
//   draw   : C_v = running float64 sum of p~ in vocabulary order,
//            y = min{v : C_v > u * W}, W the float64 total; a zero-mass
//            token is never drawn.
// The multiply-then-subtract of the logit transform must not be contracted
// into an FMA: every operation rounds on its own, as the definition states.
#pragma clang fp contract(off)

#include <float.h>
#include <limits.h>
#include <math.h>

#include "sb_device.h"
#include "sb_internal.h"

namespace sb {
namespace {

constexpr int kWalkThreads = 1024;
constexpr int kWaves = kWalkThreads / 64;

__device__ __forceinline__ double wave_sum(double v) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

__device__ __forceinline__ int wave_min(int v) {
  for (int o = 32; o > 0; o >>= 1) v = min(v, __shfl_xor(v, o, 64));
  return v;
}

__device__ __forceinline__ int wave_max(int v) {
  for (int o = 32; o > 0; o >>= 1) v = max(v, __shfl_xor(v, o, 64));
  return v;
}

// Block-wide reductions for blockDim.x == nthreads (multiple of 64).
template <int NW>
__device__ double block_sum(double v, double *red) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  v = wave_sum(v);
  if (lane == 0) red[w] = v;
  __syncthreads();
  double t = 0.0;
  if (w == 0) {
    t = lane < NW ? red[lane] : 0.0;
    t = wave_sum(t);
    if (lane == 0) red[NW] = t;
  }
  __syncthreads();
  t = red[NW];
  __syncthreads();
  return t;
}

template <int NW>
__device__ int block_min(int v, int *red) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  v = wave_min(v);
  if (lane == 0) red[w] = v;
  __syncthreads();
  if (w == 0) {
    int t = lane < NW ? red[lane] : INT_MAX;
    t = wave_min(t);
    if (lane == 0) red[NW] = t;
  }
  __syncthreads();
  int r = red[NW];
  __syncthreads();
  return r;
}

template <int NW>
__device__ int block_max(int v, int *red) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  v = wave_max(v);
  if (lane == 0) red[w] = v;
  __syncthreads();
  if (w == 0) {
    int t = lane < NW ? red[lane] : INT_MIN;
    t = wave_max(t);
    if (lane == 0) red[NW] = t;
  }
  __syncthreads();
  int r = red[NW];
  __syncthreads();
  return r;
}

// A target distribution p~: either a logits row with its statistics, or a
// residual r in the workspace with its mass Z (p~(v) = r_v / Z, the
// normalisation done element by element as it is read).
struct Dist {
  const float *l;
  float inv_t;
  float zmax;
  double total;
  int argmax;
  int greedy;
  const double *arr;  // non-null: residual array
  double zdiv;

  // p~(v), divided exactly (used for the accept ratio of a single token)
  __device__ __forceinline__ double at(int v) const {
    if (arr) return arr[v] / zdiv;
    if (greedy) return v == argmax ? 1.0 : 0.0;
    float z = l[v] * inv_t;
    float e = expf(z - zmax);
    return (double)e / total;
  }
  // 1 / (total or Z): vocabulary passes multiply by it instead of dividing
  // every element (an fp64 division is dozens of instructions); the values
  // differ from at() by at most an ulp
  __device__ __forceinline__ double recip() const { return 1.0 / (arr ? zdiv : total); }
  __device__ __forceinline__ double at_fast(int v, double rcp) const {
    if (arr) return arr[v] * rcp;
    if (greedy) return v == argmax ? 1.0 : 0.0;
    float z = l[v] * inv_t;
    float e = expf(z - zmax);
    return (double)e * rcp;
  }
};

// p~ at K tokens v[k] (invalid: v outside [0, vocab), reads as 0), the loads
// of all K issued together through wave-uniform buffer descriptors (no
// branch per element), then converted as at_fast() does.
template <int K>
__device__ __forceinline__ void load_p(const Dist &d, const int (&v)[K], int vocab, double rcp,
                                       double (&out)[K]) {
  if (d.arr) {
    const __amdgpu_buffer_rsrc_t rs = uniform_rsrc(d.arr, vocab * 8);
    uint32_t lo[K], hi[K];
#pragma unroll
    for (int k = 0; k < K; ++k) {
      const int off = (v[k] >= 0 && v[k] < vocab) ? v[k] * 8 : vocab * 8;
      lo[k] = __builtin_amdgcn_raw_buffer_load_b32(rs, off, 0, 0);
      hi[k] = __builtin_amdgcn_raw_buffer_load_b32(rs, off + 4, 0, 0);
    }
#pragma unroll
    for (int k = 0; k < K; ++k)
      out[k] = __builtin_bit_cast(double, ((uint64_t)hi[k] << 32) | lo[k]) * rcp;
  } else if (d.greedy) {
#pragma unroll
    for (int k = 0; k < K; ++k) out[k] = v[k] == d.argmax ? 1.0 : 0.0;
  } else {
    const __amdgpu_buffer_rsrc_t rs = uniform_rsrc(d.l, vocab * 4);
    float raw[K];
#pragma unroll
    for (int k = 0; k < K; ++k) {
      const int off = (v[k] >= 0 && v[k] < vocab) ? v[k] * 4 : vocab * 4;
      raw[k] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rs, off, 0, 0));
    }
#pragma unroll
    for (int k = 0; k < K; ++k) {
      const float z = raw[k] * d.inv_t;
      const double p = (double)expf(z - d.zmax) * rcp;
      out[k] = (v[k] >= 0 && v[k] < vocab) ? p : 0.0;
    }
  }
}

// p~ at the 8 consecutive tokens e0 .. e0 + 7 (e0 a multiple of 8, vocab a
// multiple of 8, so the 8 are all in range when e0 is), loaded as 16-byte
// words: a lane's 8 neighbours cost 2 (logits) or 4 (residual) loads
// instead of 8.  Converted exactly as load_p converts; !valid reads 0.
__device__ __forceinline__ void load_p8(const Dist &d, int e0, bool valid, int vocab, double rcp,
                                        double (&out)[8]) {
  if (d.arr) {
    const __amdgpu_buffer_rsrc_t rs = uniform_rsrc(d.arr, vocab * 8);
    const int off = valid ? e0 * 8 : vocab * 8;
    u32x4 w[4];
#pragma unroll
    for (int k = 0; k < 4; ++k)
      w[k] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rs, off + 16 * k, 0, 0));
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      out[2 * k] = __builtin_bit_cast(double, ((uint64_t)w[k][1] << 32) | w[k][0]) * rcp;
      out[2 * k + 1] = __builtin_bit_cast(double, ((uint64_t)w[k][3] << 32) | w[k][2]) * rcp;
    }
  } else if (d.greedy) {
#pragma unroll
    for (int e = 0; e < 8; ++e) out[e] = valid && e0 + e == d.argmax ? 1.0 : 0.0;
  } else {
    const __amdgpu_buffer_rsrc_t rs = uniform_rsrc(d.l, vocab * 4);
    const int off = valid ? e0 * 4 : vocab * 4;
    float raw[8];
#pragma unroll
    for (int k = 0; k < 2; ++k) {
      const f32x4 v = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(rs, off + 16 * k, 0, 0));
#pragma unroll
      for (int e = 0; e < 4; ++e) raw[4 * k + e] = v[e];
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float z = raw[e] * d.inv_t;
      const double p = (double)expf(z - d.zmax) * rcp;
      out[e] = valid ? p : 0.0;
    }
  }
}

__device__ __forceinline__ Dist row_dist(const float *l, const sb_row_stats &st, float inv_t,
                                         int greedy) {
  Dist d;
  d.l = l;
  d.inv_t = inv_t;
  d.zmax = st.zmax;
  d.total = st.total;
  d.argmax = st.argmax;
  d.greedy = greedy;
  d.arr = nullptr;
  d.zdiv = 1.0;
  return d;
}

struct Shared {
  double red[kWaves + 1];
  int ired[kWaves + 1];
  int decision;
  double z;
  double rcap;  // residual at the token a pass was asked to capture
};

// Elements of a vocabulary pass handled per thread per batch: their loads are
// issued together so a batch costs one memory latency.
constexpr int kBatch = 16;

// After candidate with draft row q is rejected: r = max(0, p~ - q) into
// dst; returns Z = sum r (all threads).  The new p~ is r / Z.  r at token
// xcap (the next candidate's, or -1) is also left in sh.rcap, so the next
// test needs no memory round trip.
__device__ double residual_pass(const Dist &cur, const float *q, int vocab, double *dst,
                                int xcap, Shared &sh) {
  double part = 0.0;
  const double rcp = cur.recip();
  const __amdgpu_buffer_rsrc_t qrs = uniform_rsrc(q, vocab * 4);
  for (int v0 = threadIdx.x; v0 < vocab; v0 += kBatch * kWalkThreads) {
    int vv[kBatch];
    float qv[kBatch];
    double pv[kBatch];
#pragma unroll
    for (int j = 0; j < kBatch; ++j) {
      vv[j] = v0 + j * kWalkThreads;
      qv[j] = __builtin_bit_cast(
          float, __builtin_amdgcn_raw_buffer_load_b32(qrs, (vv[j] < vocab ? vv[j] : vocab) * 4, 0, 0));
    }
    load_p<kBatch>(cur, vv, vocab, rcp, pv);
#pragma unroll
    for (int j = 0; j < kBatch; ++j) {
      const int v = v0 + j * kWalkThreads;
      double r = pv[j] - (double)qv[j];
      r = r > 0.0 ? r : 0.0;
      if (v < vocab) {
        dst[v] = r;
        part += r;
        if (v == xcap) sh.rcap = r;
      }
    }
  }
  return block_sum<kWaves>(part, sh.red);
}

// Inverse-CDF draw from p~ with uniform u (all threads return the token).
// Each wave owns a contiguous segment of the vocabulary.  Pass 1 sums the
// segments.  Pass 2 walks its segment in blocks of 512: lane l holds the 8
// consecutive elements 8l .. 8l + 7 of the block, one 64-lane inclusive scan
// of the lane sums gives each lane's prefix, the first lane whose range
// crosses u * W finds the exact token in its 8 elements.
__device__ int draw_pass(const Dist &d, float u, int vocab, Shared &sh) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int seg = ((vocab + kWaves - 1) / kWaves + 511) & ~511;
  const int lo = w * seg;
  const int hi = min(vocab, lo + seg);
  const double rcp = d.recip();
  double part = 0.0;
  for (int v0 = lo + lane; v0 < hi; v0 += 64 * kBatch) {
    int vv[kBatch];
    double x[kBatch];
#pragma unroll
    for (int j = 0; j < kBatch; ++j) vv[j] = v0 + 64 * j < hi ? v0 + 64 * j : -1;
    load_p<kBatch>(d, vv, vocab, rcp, x);
#pragma unroll
    for (int j = 0; j < kBatch; ++j) part += x[j];
  }
  part = wave_sum(part);
  if (lane == 0) sh.red[w] = part;
  __syncthreads();
  if (threadIdx.x == 0) {
    double run = 0.0;
    for (int i = 0; i < kWaves; ++i) {
      const double t = sh.red[i];
      sh.red[i] = run;  // exclusive prefix of wave i
      run += t;
    }
    sh.red[kWaves] = run;  // W
  }
  __syncthreads();
  const double base = sh.red[w];
  const double W = sh.red[kWaves];
  const double thr = (double)u * W;
  int cand = INT_MAX;
  double run = base;
  // skip whole segments that end below the threshold (their total is known)
  const double seg_end = (w + 1 < kWaves) ? sh.red[w + 1] : W;
  if (lo < hi && seg_end > thr) {
    for (int b0 = lo; b0 < hi && cand == INT_MAX; b0 += 512) {
      const int e0 = b0 + 8 * lane;
      double x[8];
      double ls = 0.0;
      if ((vocab & 7) == 0) {
        load_p8(d, e0, e0 < hi, vocab, rcp, x);
      } else {
        int vv[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) vv[e] = e0 + e < hi ? e0 + e : -1;
        load_p<8>(d, vv, vocab, rcp, x);
      }
#pragma unroll
      for (int e = 0; e < 8; ++e) ls += x[e];
      double inc = ls;
      for (int o = 1; o < 64; o <<= 1) {
        const double y = __shfl_up(inc, o, 64);
        if (lane >= o) inc += y;
      }
      const double lane_start = run + (inc - ls);
      const unsigned long long hit = __ballot(e0 < hi && lane_start + ls > thr);
      if (hit) {
        const int first = __ffsll((long long)hit) - 1;
        // the crossing lane finds the token among its 8 elements (its range
        // crosses, so one of them does unless rounding says otherwise; then
        // its last valid element)
        int found = INT_MAX;
        if (lane == first) {
          double c = lane_start;
          found = min(e0 + 7, hi - 1);
          for (int e = 0; e < 8; ++e) {
            c += x[e];
            if (e0 + e < hi && c > thr) {
              found = e0 + e;
              break;
            }
          }
        }
        cand = __shfl(found, first, 64);
      }
      run += __shfl(inc, 63, 64);
    }
  }
  int y = block_min<kWaves>(cand, sh.ired);
  if (y == INT_MAX) {
    // rounding left no crossing: the last token with positive mass
    int lp = -1;
    for (int v = threadIdx.x; v < vocab; v += kWalkThreads)
      if (d.at_fast(v, rcp) > 0.0) lp = v;
    y = block_max<kWaves>(lp, sh.ired);
    if (y < 0) y = vocab - 1;
  }
  return y;
}

// Algorithm 1 at one node.  Candidate i: token tok(i), draft row q(i),
// uniform u(i).  Returns the accepted candidate index or -1; on -1, *cur
// holds the final residual.  ws0/ws1 are two float64 [vocab] buffers.
template <class Cand>
__device__ int node_select(Dist *cur, const Cand &cand, int n_cand, int vocab, double *ws0,
                           double *ws1, int *flags, int *nrej, Shared &sh) {
  bool captured = false;  // p~(tok(i)) is sh.rcap / cur->zdiv
  for (int i = 0; i < n_cand; ++i) {
    if (threadIdx.x == 0) {
      const int x = cand.tok(i);
      double ratio = 0.0;  // a token id outside the vocabulary is rejected
      if (x >= 0 && x < vocab) {
        // q(x) gathered up front; p~(x) gathered up front while p~ is still
        // the row itself, else captured by the last residual pass
        const double qx = (double)cand.qx(i);
        if (qx == 0.0) *flags |= SB_FLAG_QZERO;
        const double px = !cur->arr ? cand.px(i) : captured ? sh.rcap / cur->zdiv : cur->at(x);
        ratio = px / qx;
      } else {
        *flags |= SB_FLAG_QZERO;
      }
      sh.decision = ((double)cand.u(i) < ratio) ? 1 : 0;
    }
    __syncthreads();
    const int acc = sh.decision;
    __syncthreads();
    if (acc) return i;
    ++*nrej;
    double *dst = (cur->arr == ws0) ? ws1 : ws0;
    const int xn = i + 1 < n_cand ? cand.tok(i + 1) : -1;
    const int xcap = xn >= 0 && xn < vocab ? xn : -1;
    double Z = residual_pass(*cur, cand.q(i), vocab, dst, xcap, sh);
    captured = false;
    if (Z > 0.0) {
      cur->arr = dst;
      cur->zdiv = Z;
      captured = xcap >= 0;
    } else if (threadIdx.x == 0) {
      *flags |= SB_FLAG_ZERO_RESIDUAL;
    }
  }
  return -1;
}

// Candidate sets.  px(i) / qx(i): the row distribution's p at the
// candidate's token and q(i) at it, valid while p~ is still that row.
struct ExplicitCands {
  const int32_t *toks;
  const float *qbase;
  const float *ubase;
  int vocab;
  const Dist *row;
  __device__ int tok(int i) const { return toks[i]; }
  __device__ const float *q(int i) const { return qbase + (size_t)i * vocab; }
  __device__ float u(int i) const { return ubase[i]; }
  __device__ double px(int i) const { return row->at(toks[i]); }
  __device__ float qx(int i) const { return q(i)[toks[i]]; }
};

struct ChildCands {
  const int16_t *kids;
  const int32_t *toks;
  const float *qbase;
  const float *ubase;
  int vocab;
  const double *pre_p;  // [row]: p of the row's parent at the row's token
  const float *pre_q;   // [row]: q of the row at its token
  __device__ int tok(int i) const { return toks[kids[i]]; }
  __device__ const float *q(int i) const { return qbase + (size_t)kids[i] * vocab; }
  __device__ float u(int i) const { return ubase[kids[i]]; }
  __device__ double px(int i) const { return pre_p[kids[i]]; }
  __device__ float qx(int i) const { return pre_q[kids[i]]; }
};

// ---------------------------------------------------------------------------

// One workgroup per row.  Pass 1: max of l (lowest-index argmax), max of
// z = fl32(l / T) and a NaN/+inf scan; pass 2: float64 sum of
// fl32(exp(z - zmax)).  Loads are 16-byte and independent across a thread's
// items so a pass costs about one memory latency.
// Row statistics with the whole row in registers (vocab a multiple of 4 and
// at most NB * 4096): one read of the row, the max / argmax / non-finite
// scan and the exp sum both run on the registers.
template <int NB>
__global__ __launch_bounds__(1024) void k_softmax_stats_reg(const float *__restrict__ logits,
                                                            int vocab, float inv_t, int greedy,
                                                            sb_row_stats *__restrict__ out,
                                                            const unsigned *invalid) {
  constexpr int NT = 1024, NW = NT / 64;
  __shared__ float smax[NW], szmax[NW];
  __shared__ int sarg[NW];
  __shared__ int sbad[NW];
  __shared__ double red[NW];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const int n4 = vocab >> 2;
  const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
      (void *)(logits + (size_t)blockIdx.x * vocab), 0, vocab * 4, kBufferDword3);
  f32x4 x[NB];
#pragma unroll
  for (int j = 0; j < NB; ++j) {
    const int i = threadIdx.x + j * NT;
    x[j] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(rs, i * 16, 0, 0));
  }
  float best = -INFINITY;
  int barg = INT_MAX;
  float zbest = -INFINITY;
  int bad = 0;
#pragma unroll
  for (int j = 0; j < NB; ++j) {
    const int i = threadIdx.x + j * NT;
    if (i < n4) {
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float v = x[j][e];
        if (isnan(v) || v == INFINITY) bad = 1;
        if (v > best) {
          best = v;
          barg = 4 * i + e;
        }
        zbest = fmaxf(zbest, v * inv_t);
      }
    }
  }
  for (int o = 32; o > 0; o >>= 1) {
    const float ob = __shfl_xor(best, o, 64);
    const int oa = __shfl_xor(barg, o, 64);
    if (ob > best || (ob == best && oa < barg)) {
      best = ob;
      barg = oa;
    }
    zbest = fmaxf(zbest, __shfl_xor(zbest, o, 64));
    bad |= __shfl_xor(bad, o, 64);
  }
  if (lane == 0) {
    smax[w] = best;
    sarg[w] = barg;
    sbad[w] = bad;
    szmax[w] = zbest;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    float b = smax[0], zb = szmax[0];
    int a = sarg[0], bd = sbad[0];
    for (int i = 1; i < NW; ++i) {
      if (smax[i] > b || (smax[i] == b && sarg[i] < a)) {
        b = smax[i];
        a = sarg[i];
      }
      zb = fmaxf(zb, szmax[i]);
      bd |= sbad[i];
    }
    smax[0] = greedy ? b : zb;
    sarg[0] = (a == INT_MAX) ? 0 : a;
    sbad[0] = bd;
  }
  __syncthreads();
  const float zmax = smax[0];
  const int arg = sarg[0];
  const int anybad = sbad[0];
  double total = 1.0;
  if (!greedy) {
    double part = 0.0;
#pragma unroll
    for (int j = 0; j < NB; ++j) {
      const int i = threadIdx.x + j * NT;
      if (i < n4)
#pragma unroll
        for (int e = 0; e < 4; ++e) part += (double)expf(x[j][e] * inv_t - zmax);
    }
    part = wave_sum(part);
    if (lane == 0) red[w] = part;
    __syncthreads();
    if (threadIdx.x == 0) {
      double t = 0.0;
      for (int i = 0; i < NW; ++i) t += red[i];
      red[0] = t;
    }
    __syncthreads();
    total = red[0];
  }
  if (threadIdx.x == 0) {
    sb_row_stats st;
    st.zmax = zmax;
    st.argmax = arg;
    // a producer that flagged the logits invalid makes the row non-finite
    st.total = (anybad || (invalid && *invalid != 0u)) ? (double)NAN : total;
    out[blockIdx.x] = st;
  }
}

// The statistics of row blockIdx.x from its groups' partials (the LM
// head's workgroups, at most 256): the largest logit and its lowest index
// over the groups, zmax = fl32(lmax / T) (rounding is monotone, so this is
// the largest scaled logit), and total = the float64 sum over groups of
// sum_g exp(m_g - zmax), m_g = fl32(lmax_g / T), in a fixed order.  A row
// with nothing above -inf has a NaN total at T > 0, as exp(-inf - -inf).
__global__ __launch_bounds__(256) void k_softmax_stats_finish(const LmPart *__restrict__ part,
                                                             int groups, float inv_t, int greedy,
                                                             sb_row_stats *__restrict__ out) {
  constexpr int NW = 256 / 64;
  __shared__ float sbest[NW];
  __shared__ int sarg[NW];
  __shared__ double red[NW + 1];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  LmPart p{-INFINITY, INT_MAX, 0.0};
  if ((int)threadIdx.x < groups) p = part[(size_t)blockIdx.x * groups + threadIdx.x];
  float best = p.lmax;
  int arg = p.arg;
  for (int o = 32; o > 0; o >>= 1) {
    const float ob = __shfl_xor(best, o, 64);
    const int oa = __shfl_xor(arg, o, 64);
    if (ob > best || (ob == best && oa < arg)) {
      best = ob;
      arg = oa;
    }
  }
  if (lane == 0) {
    sbest[w] = best;
    sarg[w] = arg;
  }
  __syncthreads();
  best = sbest[0];
  arg = sarg[0];
  for (int i = 1; i < NW; ++i)
    if (sbest[i] > best || (sbest[i] == best && sarg[i] < arg)) {
      best = sbest[i];
      arg = sarg[i];
    }
  const float zmax = greedy ? best : best * inv_t;
  double term = p.sum;
  if (!greedy && p.sum != 0.0) term = p.sum * exp((double)(p.lmax * inv_t) - (double)zmax);
  const double s = block_sum<NW>(term, red);
  if (threadIdx.x == 0) {
    sb_row_stats st;
    st.zmax = zmax;
    st.argmax = arg == INT_MAX ? 0 : arg;
    if (greedy)
      st.total = isnan(s) ? (double)NAN : 1.0;
    else
      st.total = best == -INFINITY ? (double)NAN : s;
    out[blockIdx.x] = st;
  }
}

__global__ __launch_bounds__(1024) void k_softmax_stats(const float *__restrict__ logits,
                                                        int vocab, float inv_t, int greedy,
                                                        sb_row_stats *__restrict__ out,
                                                            const unsigned *invalid) {
  constexpr int NT = 1024, NW = NT / 64;
  __shared__ float smax[NW], szmax[NW];
  __shared__ int sarg[NW];
  __shared__ int sbad[NW];
  __shared__ double red[NW];
  const float *l = logits + (size_t)blockIdx.x * vocab;
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const bool vec = (vocab & 3) == 0;
  float best = -INFINITY;
  int barg = INT_MAX;
  float zbest = -INFINITY;
  int bad = 0;
  auto visit = [&](float x, int v) {
    if (isnan(x) || x == INFINITY) bad = 1;
    if (x > best) {
      best = x;
      barg = v;
    }
    zbest = fmaxf(zbest, x * inv_t);
  };
  if (vec) {
    const float4 *l4 = (const float4 *)l;
    const int n4 = vocab >> 2;
    for (int i0 = threadIdx.x; i0 < n4; i0 += 4 * NT) {
      float4 x[4];
#pragma unroll
      for (int j = 0; j < 4; ++j)
        x[j] = (i0 + j * NT < n4) ? l4[i0 + j * NT] : make_float4(-INFINITY, -INFINITY, -INFINITY, -INFINITY);
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int i = i0 + j * NT;
        if (i < n4) {
          visit(x[j].x, 4 * i);
          visit(x[j].y, 4 * i + 1);
          visit(x[j].z, 4 * i + 2);
          visit(x[j].w, 4 * i + 3);
        }
      }
    }
  } else {
    for (int v = threadIdx.x; v < vocab; v += NT) visit(l[v], v);
  }
  for (int o = 32; o > 0; o >>= 1) {
    const float ob = __shfl_xor(best, o, 64);
    const int oa = __shfl_xor(barg, o, 64);
    if (ob > best || (ob == best && oa < barg)) {
      best = ob;
      barg = oa;
    }
    zbest = fmaxf(zbest, __shfl_xor(zbest, o, 64));
    bad |= __shfl_xor(bad, o, 64);
  }
  if (lane == 0) {
    smax[w] = best;
    sarg[w] = barg;
    sbad[w] = bad;
    szmax[w] = zbest;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    float b = smax[0], zb = szmax[0];
    int a = sarg[0], bd = sbad[0];
    for (int i = 1; i < NW; ++i) {
      if (smax[i] > b || (smax[i] == b && sarg[i] < a)) {
        b = smax[i];
        a = sarg[i];
      }
      zb = fmaxf(zb, szmax[i]);
      bd |= sbad[i];
    }
    smax[0] = greedy ? b : zb;
    sarg[0] = (a == INT_MAX) ? 0 : a;
    sbad[0] = bd;
  }
  __syncthreads();
  const float zmax = smax[0];
  const int arg = sarg[0];
  const int anybad = sbad[0];
  double total = 1.0;
  if (!greedy) {
    double part = 0.0;
    if (vec) {
      const float4 *l4 = (const float4 *)l;
      const int n4 = vocab >> 2;
      for (int i0 = threadIdx.x; i0 < n4; i0 += 4 * NT) {
        float4 x[4];
#pragma unroll
        for (int j = 0; j < 4; ++j)
          x[j] = (i0 + j * NT < n4) ? l4[i0 + j * NT] : make_float4(-INFINITY, -INFINITY, -INFINITY, -INFINITY);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          part += (double)expf(x[j].x * inv_t - zmax);
          part += (double)expf(x[j].y * inv_t - zmax);
          part += (double)expf(x[j].z * inv_t - zmax);
          part += (double)expf(x[j].w * inv_t - zmax);
        }
      }
    } else {
      for (int v = threadIdx.x; v < vocab; v += NT) part += (double)expf(l[v] * inv_t - zmax);
    }
    part = wave_sum(part);
    if (lane == 0) red[w] = part;
    __syncthreads();
    if (threadIdx.x == 0) {
      double t = 0.0;
      for (int i = 0; i < NW; ++i) t += red[i];
      red[0] = t;
    }
    __syncthreads();
    total = red[0];
  }
  if (threadIdx.x == 0) {
    sb_row_stats st;
    st.zmax = zmax;
    st.argmax = arg;
    // a producer that flagged the logits invalid makes the row non-finite
    st.total = (anybad || (invalid && *invalid != 0u)) ? (double)NAN : total;
    out[blockIdx.x] = st;
  }
}

__global__ __launch_bounds__(kWalkThreads) void k_walk(int vocab, TreeArg tree,
                                                       const int32_t *__restrict__ tokens,
                                                       const float *__restrict__ logits,
                                                       const sb_row_stats *__restrict__ stats,
                                                       float inv_t, int greedy,
                                                       const float *__restrict__ q,
                                                       const float *__restrict__ u,
                                                       sb_step_result *__restrict__ result,
                                                       double *__restrict__ ws) {
  __shared__ Shared sh;
  __shared__ int16_t kids[SB_MAX_ROWS];
  __shared__ int16_t path[SB_MAX_ROWS];
  __shared__ int nk;
  __shared__ int s_flags;
  __shared__ sb_row_stats s_st[SB_MAX_ROWS];
  __shared__ double s_px[SB_MAX_ROWS];
  __shared__ float s_qx[SB_MAX_ROWS];
  __shared__ int16_t s_par[SB_MAX_ROWS];
  __shared__ unsigned long long s_kmask[(SB_MAX_ROWS + 63) / 64];
  __shared__ int32_t s_tok[SB_MAX_ROWS];
  __shared__ float s_u[SB_MAX_ROWS];
  __shared__ int s_first[SB_MAX_ROWS];  // lowest-index child of a row (INT_MAX: none)
  __shared__ int s_node, s_plen;
  const int n = tree.n;
  double *ws0 = ws;
  double *ws1 = ws + vocab;
  if (threadIdx.x == 0) s_flags = 0;
  // the tree (kernel arguments: every dynamically indexed read is a memory
  // access) and every row's statistics into LDS, then in parallel every
  // row's test values: p of its parent at its token and q at its token (the
  // walk's chain tests then read LDS instead of paying a memory round trip
  // each)
  if ((int)threadIdx.x < n) {
    s_par[threadIdx.x] = tree.parent[threadIdx.x];
    s_st[threadIdx.x] = stats[threadIdx.x];
    s_tok[threadIdx.x] = tokens[threadIdx.x];
    s_u[threadIdx.x] = u[threadIdx.x];
  }
  if ((int)threadIdx.x < SB_MAX_ROWS) s_first[threadIdx.x] = INT_MAX;
  __syncthreads();
  // first children: the candidates tried first at every node
  if ((int)threadIdx.x >= 1 && (int)threadIdx.x < n) atomicMin(&s_first[s_par[threadIdx.x]], (int)threadIdx.x);
  if ((int)threadIdx.x < n && isnan(s_st[threadIdx.x].total)) atomicOr(&s_flags, SB_FLAG_NONFINITE);
  if ((int)threadIdx.x >= 1 && (int)threadIdx.x < n) {
    const int i = threadIdx.x;
    const int x = tokens[i];
    const int par = s_par[i];
    double px = 0.0;
    float qx = 0.0f;
    if (x >= 0 && x < vocab) {
      px = row_dist(logits + (size_t)par * vocab, s_st[par], inv_t, greedy).at(x);
      qx = q[(size_t)i * vocab + x];
    }
    s_px[i] = px;
    s_qx[i] = qx;
  }
  __syncthreads();
  int flags = 0;  // thread 0 accumulates
  int nrej = 0;
  // Accept chain: while every node's first candidate is accepted against
  // the node's own row (no residual yet), the tests read LDS only, so one
  // thread walks them with no barrier per level.  The walk below resumes at
  // the first node whose first candidate fails (it repeats that test and
  // goes on with the residuals) or at the leaf reached.
  if (threadIdx.x == 0) {
    int nd = 0, pl = 1;
    path[0] = 0;
    for (;;) {
      const int c = s_first[nd];
      if (c == INT_MAX) break;
      const int x = s_tok[c];
      double ratio = 0.0;
      if (x >= 0 && x < vocab) {
        const double qx = (double)s_qx[c];
        if (qx == 0.0) flags |= SB_FLAG_QZERO;
        ratio = s_px[c] / qx;
      } else {
        flags |= SB_FLAG_QZERO;
      }
      if (!((double)s_u[c] < ratio)) break;
      path[pl++] = (int16_t)c;
      nd = c;
    }
    s_node = nd;
    s_plen = pl;
  }
  __syncthreads();
  int node = s_node;
  int plen = s_plen;
  Dist cur = row_dist(logits + (size_t)node * vocab, s_st[node], inv_t, greedy);
  int y = 0;
  int bonus = 0;
  for (;;) {
    // the children of `node` in index order: one ballot per wave over the
    // rows, then thread 0 lists the set bits
    {
      const int j = threadIdx.x;
      const unsigned long long m = __ballot(j > node && j < n && s_par[j] == node);
      if ((j & 63) == 0 && j < SB_MAX_ROWS) s_kmask[j >> 6] = m;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
      int c = 0;
      for (int wv = 0; wv * 64 < n; ++wv) {
        unsigned long long m = s_kmask[wv];
        while (m) {
          kids[c++] = (int16_t)(wv * 64 + __ffsll((long long)m) - 1);
          m &= m - 1;
        }
      }
      nk = c;
    }
    __syncthreads();
    const int nkids = nk;
    if (nkids == 0) {
      bonus = 1;
      break;
    }
    ChildCands cc{kids, s_tok, q, s_u, vocab, s_px, s_qx};
    const int acc = node_select(&cur, cc, nkids, vocab, ws0, ws1, &flags, &nrej, sh);
    if (acc >= 0) {
      node = kids[acc];
      __syncthreads();
      if (threadIdx.x == 0) path[plen] = (int16_t)node;
      ++plen;
      cur = row_dist(logits + (size_t)node * vocab, s_st[node], inv_t, greedy);
      continue;
    }
    break;
  }
  // the bonus token from an accepted leaf's p, or the residual's draw
  y = draw_pass(cur, u[0], vocab, sh);
  __syncthreads();
  if (threadIdx.x == 0) {
    int branch = -1;
    if (plen > 1) {
      int ord = 0;
      for (int j = 1; j < path[1]; ++j)
        if (s_par[j] == 0) ++ord;
      branch = ord;
    }
    result->n_accepted = plen - 1;
    result->branch = branch;
    result->next_token = y;
    result->path_len = plen;
    result->flags = flags | s_flags;
    result->n_rejected = nrej;
    result->bonus = bonus;
    result->reserved = 0;
  }
  for (int j = threadIdx.x; j < SB_MAX_ROWS; j += kWalkThreads)
    result->path[j] = j < plen ? (int32_t)path[j] : -1;
}

__global__ __launch_bounds__(kWalkThreads) void k_select(int vocab, const float *__restrict__ lrow,
                                                         const sb_row_stats *__restrict__ st,
                                                         float inv_t, int greedy, int n_cand,
                                                         const int32_t *__restrict__ ctoks,
                                                         const float *__restrict__ q,
                                                         const float *__restrict__ u,
                                                         int32_t *__restrict__ out,
                                                         double *__restrict__ ws) {
  __shared__ Shared sh;
  int flags = 0, nrej = 0;
  const sb_row_stats s0 = st[0];
  if (isnan(s0.total)) flags |= SB_FLAG_NONFINITE;
  Dist cur = row_dist(lrow, s0, inv_t, greedy);
  ExplicitCands ec{ctoks, q, u, vocab, &cur};
  const int acc = node_select(&cur, ec, n_cand, vocab, ws, ws + vocab, &flags, &nrej, sh);
  int tok;
  if (acc >= 0) {
    tok = ctoks[acc];
  } else {
    tok = draw_pass(cur, u[n_cand], vocab, sh);
  }
  if (threadIdx.x == 0) {
    out[0] = acc;
    out[1] = tok;
    out[2] = flags;
  }
}

// The draft's rows (the draft side of a round): q(v) = float32(p(v)) of a
// logits row at T, written out as the row verification later reads as q,
// and the token drawn from those float32 values: their float64 running sum
// in vocabulary order, the first v whose sum exceeds u * W.  T = 0: q is
// one-hot at the row's argmax, which is the token.
//   k_draft_q:    grid (blocks of kDraftSpan tokens, rows); writes q and the
//                 float64 sum of each block's q to the workspace;
//   k_draft_draw: one workgroup per row; the crossing block from the block
//                 sums, then the token from that block's q.
constexpr int kDraftThreads = 256;
constexpr int kDraftSpan = kDraftThreads * 8;

__device__ __forceinline__ float draft_qv(float raw, float inv_t, float zmax, double total) {
  const float z = raw * inv_t;
  const float e = expf(z - zmax);
  return (float)((double)e / total);
}

__global__ __launch_bounds__(kDraftThreads) void k_draft_q(int vocab, int vec8, DraftRows rows,
                                                           const float *__restrict__ logits,
                                                           const sb_row_stats *__restrict__ stats,
                                                           float inv_t, int greedy,
                                                           float *__restrict__ q,
                                                           double *__restrict__ bsum) {
  __shared__ double red[kDraftThreads / 64];
  const int i = blockIdx.y, blk = blockIdx.x, nblk = gridDim.x;
  const int src = rows.src[i], dst = rows.dst[i];
  const float *l = logits + (size_t)src * vocab;
  const sb_row_stats st = stats[src];
  float *qr = q + (size_t)dst * vocab;
  // thread t: the 8 consecutive tokens v0 .. v0 + 7 of the block (whole
  // 16-byte pairs when vocab % 8 == 0 and the rows are 16-byte aligned)
  const int v0 = blk * kDraftSpan + (int)threadIdx.x * 8;
  float raw[8];
  if (vec8 && v0 < vocab) {
    const f32x4 a = *(const f32x4 *)(l + v0), b = *(const f32x4 *)(l + v0 + 4);
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      raw[e] = a[e];
      raw[4 + e] = b[e];
    }
  } else {
#pragma unroll
    for (int e = 0; e < 8; ++e) raw[e] = v0 + e < vocab ? l[v0 + e] : 0.0f;
  }
  float f[8];
  double part = 0.0;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const int v = v0 + e;
    f[e] = greedy ? (v == st.argmax ? 1.0f : 0.0f) : draft_qv(raw[e], inv_t, st.zmax, st.total);
    if (v < vocab) part += (double)f[e];
  }
  if (vec8 && v0 < vocab) {
    *(f32x4 *)(qr + v0) = f32x4{f[0], f[1], f[2], f[3]};
    *(f32x4 *)(qr + v0 + 4) = f32x4{f[4], f[5], f[6], f[7]};
  } else {
#pragma unroll
    for (int e = 0; e < 8; ++e)
      if (v0 + e < vocab) qr[v0 + e] = f[e];
  }
  part = wave_sum(part);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = part;
  __syncthreads();
  if (threadIdx.x == 0) {
    double t = red[0];
    for (int w = 1; w < kDraftThreads / 64; ++w) t += red[w];
    bsum[(size_t)i * nblk + blk] = t;
  }
}

// Inclusive 64-lane scan of a double.
__device__ __forceinline__ double wave_scan(double x) {
  const int lane = threadIdx.x & 63;
  for (int o = 1; o < 64; o <<= 1) {
    const double y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  return x;
}

__global__ __launch_bounds__(kDraftThreads) void k_draft_draw(int vocab, int nblk, DraftRows rows,
                                                              const sb_row_stats *__restrict__ stats,
                                                              int greedy, const float *__restrict__ u,
                                                              int32_t *__restrict__ tokens,
                                                              const float *__restrict__ q,
                                                              const double *__restrict__ bsum,
                                                              float *__restrict__ conf) {
  __shared__ double s_base, s_thr, wsum[kDraftThreads / 64];
  __shared__ int s_blk, s_tok;
  const int i = blockIdx.x;
  const int src = rows.src[i], dst = rows.dst[i];
  if (greedy) {
    if (threadIdx.x == 0) {
      tokens[dst] = stats[src].argmax;
      if (conf) conf[i] = 1.0f;
    }
    return;
  }
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  const double *bs = bsum + (size_t)i * nblk;
  // wave 0: lane l sums the block sums l*per .. l*per + per - 1 in order,
  // scans the lane sums, and finds the first block whose running sum
  // exceeds u * W (else the last block with mass)
  if (w == 0) {
    const int per = (nblk + 63) / 64;
    double ls = 0.0;
    for (int j = 0; j < per; ++j) {
      const int b = lane * per + j;
      if (b < nblk) ls += bs[b];
    }
    const double inc = wave_scan(ls);
    const double W = __shfl(inc, 63, 64);
    const double thr = (double)u[i] * W;
    const unsigned long long hit = __ballot(ls > 0.0 && inc > thr);
    int sel_lane;
    if (hit) {
      sel_lane = __ffsll((long long)hit) - 1;
    } else {
      const unsigned long long pos = __ballot(ls > 0.0);
      sel_lane = pos ? 63 - __clzll((long long)pos) : 0;
    }
    if (lane == sel_lane) {
      double run = inc - ls;
      int blk = -1, last = -1;
      double base_at = run, base_last = run;
      for (int j = 0; j < per; ++j) {
        const int b = lane * per + j;
        if (b >= nblk) break;
        const double x = bs[b];
        if (x > 0.0) {
          last = b;
          base_last = run;
          if (blk < 0 && run + x > thr) {
            blk = b;
            base_at = run;
          }
        }
        run += x;
      }
      if (blk < 0) {
        blk = last < 0 ? 0 : last;
        base_at = base_last;
      }
      s_blk = blk;
      s_base = base_at;
      s_thr = thr;
    }
  }
  __syncthreads();
  // the crossing block: thread t holds its 8 consecutive values, a block-wide
  // scan of the thread sums finds the thread, that thread finds the token
  const int blk = s_blk;
  const double thr = s_thr - s_base;
  const int v0 = blk * kDraftSpan + (int)threadIdx.x * 8;
  const float *qr = q + (size_t)dst * vocab;
  double x[8], ts = 0.0;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    x[e] = v0 + e < vocab ? (double)qr[v0 + e] : 0.0;
    ts += x[e];
  }
  const double inc = wave_scan(ts);
  if (lane == 63) wsum[w] = inc;
  if (threadIdx.x == 0) s_tok = INT_MAX;
  __syncthreads();
  double off = 0.0;
  for (int k = 0; k < w; ++k) off += wsum[k];
  const double start = off + inc - ts;
  const unsigned long long hit = __ballot(ts > 0.0 && start + ts > thr);
  int found = INT_MAX;
  if (hit && lane == __ffsll((long long)hit) - 1) {
    double c = start;
    for (int e = 0; e < 8; ++e) {
      c += x[e];
      if (x[e] > 0.0 && c > thr) {
        found = v0 + e;
        break;
      }
    }
    if (found == INT_MAX)  // rounding: the thread's last token with mass
      for (int e = 0; e < 8; ++e)
        if (x[e] > 0.0) found = v0 + e;
  }
  if (found != INT_MAX) atomicMin(&s_tok, found);
  __syncthreads();
  if (threadIdx.x == 0) {
    int y = s_tok;
    if (y == INT_MAX) {
      // rounding left no crossing in the block: its last token with mass
      for (int v = min(vocab, (blk + 1) * kDraftSpan) - 1; v >= blk * kDraftSpan; --v)
        if (qr[v] > 0.0f) {
          y = v;
          break;
        }
      if (y == INT_MAX) y = stats[src].argmax;
    }
    tokens[dst] = y;
    if (conf) conf[i] = qr[y];  // the drawn token's own probability
  }
}

// A chain draft's q row conditioned on confidence, in place: q(v) / q(C)
// on C = {v : q(v) >= eps} (float32 comparisons), zero elsewhere, with q(C)
// the float64 sum of C's float32 values and each quotient rounded once to
// float32.  A row with no confident token is left all zero.
__global__ __launch_bounds__(kWalkThreads) void k_confident_row(float *q, int vocab, float eps) {
  __shared__ double red[kWaves + 1];
  double part = 0.0;
  for (int v = threadIdx.x; v < vocab; v += kWalkThreads) {
    const float x = q[v];
    if (x >= eps) part += (double)x;
  }
  const double mass = block_sum<kWaves>(part, red);
  for (int v = threadIdx.x; v < vocab; v += kWalkThreads) {
    const float x = q[v];
    q[v] = x >= eps && mass > 0.0 ? (float)((double)x / mass) : 0.0f;
  }
}

}  // namespace

hipError_t launch_confident_row(float *q, int vocab, float eps, hipStream_t s) {
  hipLaunchKernelGGL(k_confident_row, dim3(1), dim3(kWalkThreads), 0, s, q, vocab, eps);
  return hipGetLastError();
}

size_t sample_ws_bytes(int vocab) { return (size_t)2 * (size_t)vocab * sizeof(double); }

static inline void temp_args(float temperature, float *inv_t, int *greedy) {
  *greedy = temperature <= 0.0f ? 1 : 0;
  *inv_t = *greedy ? 1.0f : 1.0f / temperature;
}

hipError_t launch_softmax_stats(int vocab, int n_rows, const float *logits, float temperature,
                                sb_row_stats *stats, hipStream_t s, const unsigned *invalid) {
  float inv_t;
  int greedy;
  temp_args(temperature, &inv_t, &greedy);
  const int nb = (vocab + 4095) / 4096;  // float4 per thread with the row in registers
  if ((vocab & 3) == 0 && nb <= 16) {
#define SB_NB(k)                                                                                  \
  if (nb <= k) {                                                                                  \
    hipLaunchKernelGGL(k_softmax_stats_reg<k>, dim3(n_rows), dim3(1024), 0, s, logits, vocab,     \
                       inv_t, greedy, stats, invalid);                                            \
    return hipGetLastError();                                                                     \
  }
    SB_NB(1) SB_NB(2) SB_NB(4) SB_NB(8) SB_NB(16)
#undef SB_NB
  }
  hipLaunchKernelGGL(k_softmax_stats, dim3(n_rows), dim3(1024), 0, s, logits, vocab, inv_t, greedy,
                     stats, invalid);
  return hipGetLastError();
}

hipError_t launch_stats_finish(const LmPart *part, int groups, int n_rows, float temperature,
                               sb_row_stats *stats, hipStream_t s) {
  if (groups < 1 || groups > 256 || n_rows < 1) return hipErrorInvalidValue;
  float inv_t;
  int greedy;
  temp_args(temperature, &inv_t, &greedy);
  hipLaunchKernelGGL(k_softmax_stats_finish, dim3(n_rows), dim3(256), 0, s, part, groups, inv_t,
                     greedy, stats);
  return hipGetLastError();
}

hipError_t launch_walk(int vocab, const TreeArg &tree, const int32_t *tokens, const float *logits,
                       const sb_row_stats *stats, float temperature, const float *q,
                       const float *u, sb_step_result *result, void *ws, hipStream_t s) {
  float inv_t;
  int greedy;
  temp_args(temperature, &inv_t, &greedy);
  hipLaunchKernelGGL(k_walk, dim3(1), dim3(kWalkThreads), 0, s, vocab, tree, tokens, logits, stats,
                     inv_t, greedy, q, u, result, (double *)ws);
  return hipGetLastError();
}

size_t draft_ws_bytes(int vocab, int n) {
  return (size_t)n * ((vocab + kDraftSpan - 1) / kDraftSpan) * sizeof(double);
}

hipError_t launch_draft_sample(int vocab, const DraftRows &rows, const float *logits,
                               const sb_row_stats *stats, float temperature, const float *u,
                               int32_t *tokens, float *q, void *ws, hipStream_t s, float *conf) {
  float inv_t;
  int greedy;
  temp_args(temperature, &inv_t, &greedy);
  const int nblk = (vocab + kDraftSpan - 1) / kDraftSpan;
  const int vec8 = vocab % 8 == 0 && ((uintptr_t)logits & 15) == 0 && ((uintptr_t)q & 15) == 0;
  hipLaunchKernelGGL(k_draft_q, dim3(nblk, rows.n), dim3(kDraftThreads), 0, s, vocab, vec8, rows,
                     logits, stats, inv_t, greedy, q, (double *)ws);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(k_draft_draw, dim3(rows.n), dim3(kDraftThreads), 0, s, vocab, nblk, rows,
                     stats, greedy, u, tokens, q, (const double *)ws, conf);
  return hipGetLastError();
}

hipError_t launch_select(int vocab, const float *logits_row, const sb_row_stats *stats_row,
                         float temperature, int n_cand, const int32_t *cand_tokens,
                         const float *q, const float *u, int32_t *out, void *ws, hipStream_t s) {
  float inv_t;
  int greedy;
  temp_args(temperature, &inv_t, &greedy);
  hipLaunchKernelGGL(k_select, dim3(1), dim3(kWalkThreads), 0, s, vocab, logits_row, stats_row,
                     inv_t, greedy, n_cand, cand_tokens, q, u, out, (double *)ws);
  return hipGetLastError();
}

}  // namespace sb
