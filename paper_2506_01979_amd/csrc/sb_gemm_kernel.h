// Skinny matrix-core GEMM kernel with fused epilogues (gfx950), included
// by one translation unit per epilogue kind.
//
// The verify forward multiplies n_rows (5..256) activation rows by every
// weight matrix once; the weights (13-140 GB) dominate the bytes, so the
// GEMM streams each weight tile from HBM exactly once with 16-byte loads in
// the operand order of v_mfma_f32_16x16x32_bf16 (the layout sb_pack_weight
// writes).  One workgroup per compute unit owns a range of weight tiles and
// walks K in chunks, reusing each activation fragment across all of its
// tiles.  The epilogue kind is a template parameter, so a kernel holds the
// registers of its own epilogue only.
#pragma once

#include <limits.h>
#include <math.h>

#include <hip/hip_ext.h>

#include "sb_device.h"
#include "sb_internal_fwd.h"

namespace sb {
namespace {

constexpr int kGemmThreads = 512;
constexpr int kGemmWaves = kGemmThreads / 64;

// ---------------------------------------------------------------------------
// skinny matrix-core GEMM with fused epilogues
// ---------------------------------------------------------------------------

__device__ __forceinline__ void rope_pair(float x1, float x2, float2 cs, float *o1, float *o2) {
  *o1 = x1 * cs.x - x2 * cs.y;
  *o2 = x2 * cs.x + x1 * cs.y;
}

// Four floats to bf16 (round to nearest even), as one 8-byte word.
__device__ __forceinline__ uint2 pack4_bf16(float x0, float x1, float x2, float x3) {
  return make_uint2(f2bf(x0) | ((uint32_t)f2bf(x1) << 16), f2bf(x2) | ((uint32_t)f2bf(x3) << 16));
}

// Four consecutive floats row[d .. d + 3] (d a multiple of 4), only those
// below n; one 16-byte store when the row is 16-byte aligned (n % 4 == 0).
__device__ __forceinline__ void store4f(float *row, int d, int n, const f32x4 &v) {
  if ((n & 3) == 0 && d + 3 < n) {
    *(f32x4 *)(row + d) = v;
  } else {
#pragma unroll
    for (int i = 0; i < 4; ++i)
      if (d + i < n) row[d + i] = v[i];
  }
}

// Epilogue of four finished output pairs of tile `tile`: rows p0 + i and
// p0 + 8 + i (i < 4, p0 = 0 or 4), activation row t < n_tok, values v1[i] /
// v2[i] (K range `split` of a split-K launch).
template <int EPI>
__device__ __forceinline__ void epilogue4(const GemmArgs &a, const float2 *rope, int split,
                                          int tile, int p0, int t, const f32x4 &v1,
                                          const f32x4 &v2) {
  if constexpr (EPI == EPI_QKV) {
    const int d = a.head_dim, ht = d / 16;
    const int qt = a.n_heads * ht, kt = a.n_kv * ht;
    if (tile < qt + kt) {
      // a Q / K tile holds the RoPE pairs (j, j + d/2), j = 8u .. 8u + 7
      const bool isq = tile < qt;
      const int idx = isq ? tile : tile - qt;
      const int head = idx / ht, u = idx % ht;
      const int j0 = 8 * u + p0;
      const f32x4 c01 = *(const f32x4 *)(rope + t * (d / 2) + j0);
      const f32x4 c23 = *(const f32x4 *)(rope + t * (d / 2) + j0 + 2);
      float o1[4], o2[4];
      rope_pair(v1[0], v2[0], make_float2(c01[0], c01[1]), &o1[0], &o2[0]);
      rope_pair(v1[1], v2[1], make_float2(c01[2], c01[3]), &o1[1], &o2[1]);
      rope_pair(v1[2], v2[2], make_float2(c23[0], c23[1]), &o1[2], &o2[2]);
      rope_pair(v1[3], v2[3], make_float2(c23[2], c23[3]), &o1[3], &o2[3]);
      uint16_t *dst = isq ? a.q + ((size_t)t * a.n_heads + head) * d
                          : a.kc + ((size_t)head * a.cap + a.kv_len + t) * d;
      *(uint2 *)(dst + j0) = pack4_bf16(o1[0], o1[1], o1[2], o1[3]);
      *(uint2 *)(dst + j0 + d / 2) = pack4_bf16(o2[0], o2[1], o2[2], o2[3]);
    } else {
      // V is cached transposed: [head][d][slot]
      const int idx = tile - qt - kt;
      const int head = idx / ht, u = idx % ht;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        uint16_t *col = a.vc + ((size_t)head * d + 16 * u + p0 + i) * a.cap + a.kv_len + t;
        col[0] = f2bf(v1[i]);
        col[(size_t)8 * a.cap] = f2bf(v2[i]);
      }
    }
  } else if constexpr (EPI == EPI_RESID) {
    // the projection is stored as a delta (one slice per K range); the next
    // RMSNorm adds the slices to the residual stream
    float *drow = a.h + ((size_t)split * a.n_tok + t) * a.out_rows;
    store4f(drow, tile * 16 + p0, a.out_rows, v1);
    store4f(drow, tile * 16 + p0 + 8, a.out_rows, v2);
  } else if constexpr (EPI == EPI_SWIGLU) {
    // rows p of a tile are gate rows, rows p + 8 the matching up rows;
    // silu(g) = g / (1 + e^-g) with the hardware exp2 and reciprocal (the
    // result is rounded to bf16)
    float o[4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
      o[i] = v1[i] * __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(v1[i] * -1.44269504f)) * v2[i];
    *(uint2 *)(a.act + packed_index(t, tile * 8 + p0, a.act_ks)) = pack4_bf16(o[0], o[1], o[2], o[3]);
  } else if constexpr (EPI == EPI_LOGITS) {
    float *lrow = a.logits + (size_t)t * a.out_rows;
    store4f(lrow, tile * 16 + p0, a.out_rows, v1);
    store4f(lrow, tile * 16 + p0 + 8, a.out_rows, v2);
  }
}

// Chunk-major weight-streaming GEMM.
//
// K is cut into chunks of 8 k-steps; wave w of a workgroup owns k-step
// 8c + w of every chunk c.  A workgroup owns a range of 16-row weight tiles
// (and, for split-K launches, one K range), and a wave walks its chunks in
// order: per chunk it loads its TT activation fragments once and the NT
// weight fragments of that k-step (one per tile), so each activation
// fragment feeds NT matrix-core products.  Activation re-reads from L2 are
// what limits a skinny GEMM whose waves stream one tile at a time; reusing
// them across the workgroup's tiles cuts that traffic NT-fold.  Loads run R
// chunks ahead in a register ring.  At the end the 8 waves' partial sums of
// every tile are reduced in LDS and the epilogue runs.
//
// Ring depth per (TT, NT): as deep as the 256-register budget of two waves
// per SIMD allows (ring 4R(NT+TT), accumulators 4*NT*TT, lane offsets NT+TT,
// about 48 for the rest), up to about 12 KB of weights in flight per wave
// (96 KB per compute unit: what covers the HBM latency at the per-unit
// share of the bandwidth), and at least 4 chunks.
template <int TT, int NT>
struct Ring {
  static constexpr int free_regs = 208 - TT - NT - 4 * NT * TT;
  static constexpr int r = free_regs / (4 * (NT + TT));
  static constexpr int cap = 12 / NT > 4 ? 12 / NT : 4;
  static constexpr int R = r > cap ? cap : (r < 1 ? 1 : r);
};

// LDS staging area (32 KB): the step's RoPE table (QKV), the residual rows
// and gains of the group's tiles (RESID_NORM), or the RMSNorm scales of the
// tokens (the consumer of a RESID_NORM launch).
constexpr int kStageBytes = 32768;
constexpr int kRopeLds = kStageBytes / 8;  // float2 entries
constexpr int kStageGain = 16384;          // RESID_NORM: gains (1 KB)
constexpr int kStageSq = 17408;            // RESID_NORM: per-(tile, token) sums of squares
constexpr int kStageLmSlot = 0;            // LOGITS: statistics per (part, token), 8 KB

// Workgroup barrier for LDS traffic only (does not wait for global loads).
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

typedef __attribute__((address_space(3))) void lds_void;

// RESID_NORM epilogue of four output pairs (rows p0 + i, p0 + 8 + i of the
// tile, token t): adds the projection to the residual (staged row hrow),
// stores it, packs bf16(h * gain) for the next projection and returns the
// pairs' sum of squares.
__device__ __forceinline__ float resid_norm4(const GemmArgs &a, const float *hrow,
                                             const float *gain, int tile, int p0, int t,
                                             const f32x4 &v1, const f32x4 &v2) {
  const int n = a.out_rows;
  const f32x4 h1 = *(const f32x4 *)(hrow + p0) + v1;
  const f32x4 h2 = *(const f32x4 *)(hrow + p0 + 8) + v2;
  const f32x4 g1 = *(const f32x4 *)(gain + p0);
  const f32x4 g2 = *(const f32x4 *)(gain + p0 + 8);
  float *hg = a.h + (size_t)t * n;
  const int d1 = tile * 16 + p0, d2 = d1 + 8;
  store4f(hg, d1, n, h1);
  store4f(hg, d2, n, h2);
  float sq = 0.0f;
  if (d1 + 3 < n) {
    *(uint2 *)(a.xn + packed_index(t, d1, a.xn_ks)) =
        pack4_bf16(h1[0] * g1[0], h1[1] * g1[1], h1[2] * g1[2], h1[3] * g1[3]);
    sq = (h1[0] * h1[0] + h1[1] * h1[1]) + (h1[2] * h1[2] + h1[3] * h1[3]);
  } else {
#pragma unroll
    for (int i = 0; i < 4; ++i)
      if (d1 + i < n) {
        a.xn[packed_index(t, d1 + i, a.xn_ks)] = f2bf(h1[i] * g1[i]);
        sq += h1[i] * h1[i];
      }
  }
  if (d2 + 3 < n) {
    *(uint2 *)(a.xn + packed_index(t, d2, a.xn_ks)) =
        pack4_bf16(h2[0] * g2[0], h2[1] * g2[1], h2[2] * g2[2], h2[3] * g2[3]);
    sq += (h2[0] * h2[0] + h2[1] * h2[1]) + (h2[2] * h2[2] + h2[3] * h2[3]);
  } else {
#pragma unroll
    for (int i = 0; i < 4; ++i)
      if (d2 + i < n) {
        a.xn[packed_index(t, d2 + i, a.xn_ks)] = f2bf(h2[i] * g2[i]);
        sq += h2[i] * h2[i];
      }
  }
  return sq;
}

// LOGITS with fused softmax statistics: the partial statistics of 16
// consecutive logits x[0 .. 15] of one token row, columns c0 .. c0 + 15
// (columns past the vocabulary are not logits).
__device__ __forceinline__ LmPart lm_cols(const GemmArgs &a, const float (&x)[16], int c0) {
  float best = -INFINITY;
  int arg = INT_MAX;
  bool bad = false;
  float v[16];
#pragma unroll
  for (int j = 0; j < 16; ++j) {
    v[j] = c0 + j < a.out_rows ? x[j] : -INFINITY;
    bad |= isnan(v[j]) || v[j] == INFINITY;
    const bool take = v[j] > best;  // in column order: the lowest index of the largest
    best = take ? v[j] : best;
    arg = take ? c0 + j : arg;
  }
  double sum = bad ? (double)NAN : 0.0;
  if (!bad && !a.lm_greedy && best > -INFINITY) {
    const float m = best * a.lm_inv_t;
#pragma unroll
    for (int j = 0; j < 16; ++j) sum += (double)expf(v[j] * a.lm_inv_t - m);
  }
  return LmPart{best, arg, sum};
}

// exp(x - y) for floats x <= y to about float precision: the difference is
// exact in float64; its float part goes through the float exponential and
// the remainder d - fl32(d), below half an ulp of d, through 1 + r.
// Below -104 (-inf included) the float exponential is 0; two infinities of
// one sign give NaN, as exp(inf - inf).
__device__ __forceinline__ double exp_diff(float x, float y) {
  const double d = (double)x - (double)y;
  if (d < -104.0) return 0.0;
  const float dh = (float)d;
  return (double)expf(dh) * (1.0 + (d - (double)dh));
}

// Running statistics r (sum relative to fl32(r.lmax / T)) merged with a
// partial p (sum relative to fl32(p.lmax / T)).
__device__ __forceinline__ void lm_merge(LmPart &r, const LmPart &p, float inv_t, int greedy) {
  const float old = r.lmax;
  if (p.lmax > r.lmax || (p.lmax == r.lmax && p.arg < r.arg)) {
    r.lmax = p.lmax;
    r.arg = p.arg;
  }
  if (greedy) {
    r.sum += p.sum;  // NaN marks a row with a NaN or +inf logit
    return;
  }
  if (p.sum == 0.0) return;  // nothing above -inf
  const float mo = old * inv_t, mp = p.lmax * inv_t;
  if (mp > mo)
    r.sum = r.sum * exp_diff(mo, mp) + p.sum;
  else
    r.sum += p.sum * exp_diff(mp, mo);
}

template <int EPI, int TT, int NT>
__global__ __launch_bounds__(kGemmThreads, 1) void k_gemm(GemmArgs a) {
  __shared__ f32x4 red[kGemmWaves][kRedPairs][64];
  __shared__ __attribute__((aligned(16))) char stage[kStageBytes];
  constexpr int R = Ring<TT, NT>::R;
  constexpr int TPR = kRedPairs / TT > 0 ? kRedPairs / TT : 1;  // tiles per reduction round
  // wave-uniform quantities live in scalar registers
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int ks = a.ks;
  const int S = a.split;
  // Workgroups are dispatched round-robin over the 8 XCDs (block b runs on
  // XCD b % 8).  Work unit u = (tile group, K range) is numbered XCD-major,
  // so each XCD streams one contiguous eighth of the weights: the XCDs move
  // equal bytes even when the groups' tile counts differ by one.
  const int nb = gridDim.x;
  const int u = (nb & 7) == 0 ? (blockIdx.x & 7) * (nb >> 3) + (blockIdx.x >> 3) : blockIdx.x;
  const int split = u % S, grp = u / S;
  const int t_lo = (int)(((long long)a.tiles * grp) / a.groups);
  const int t_hi = (int)(((long long)a.tiles * (grp + 1)) / a.groups);
  const int nc = ks >> 3;
  const int c_begin = (nc * split) / S;
  const int n_ch = (nc * (split + 1)) / S - c_begin;
  // Activation lanes of rows >= n_tok point past the end of the buffer and
  // read as zero; weight lanes of tiles past the group's end likewise.
  const int xbytes = ((a.n_tok + 15) >> 4) * ks * 1024;
  const __amdgpu_buffer_rsrc_t xrs =
      __builtin_amdgcn_make_buffer_rsrc((void *)a.X, 0, xbytes, kBufferDword3);
  int xvo[TT];
#pragma unroll
  for (int tt = 0; tt < TT; ++tt)
    xvo[tt] = (tt * 16 + (lane & 15)) < a.n_tok
                  ? tt * ks * 1024 + (lane & 15) * 64 + (lane >> 4) * 16
                  : xbytes;

  // Operands of the epilogue go to LDS by direct-to-LDS loads issued now (no
  // registers held; each wave instruction moves 1 KB), long before the
  // epilogue needs them.
  // QKV: the step's RoPE table (its buffer holds whole 1 KB blocks: rows
  // padded to 16).
  const bool rope_lds = EPI == EPI_QKV && a.n_tok * (a.head_dim / 2) <= kRopeLds;
  if (rope_lds) {
    const int nblk = (a.n_tok * (a.head_dim / 2) * 8 + 1023) >> 10;
    for (int b = w; b < nblk; b += kGemmWaves)
      __builtin_amdgcn_global_load_lds((const void *)((const char *)a.rope + b * 1024 + lane * 16),
                                       (lds_void *)(stage + b * 1024), 16, 0, 0);
  }
  // RESID_NORM (one pass, one reduction round): block (tile tl, token tile
  // tt) of the residual, [16 tokens][16 rows] fp32, and the group's gains.
  // Tokens >= n_tok read zero.
  if constexpr (EPI == EPI_RESID_NORM) {
    const __amdgpu_buffer_rsrc_t hrs = __builtin_amdgcn_make_buffer_rsrc(
        (void *)a.h, 0, a.n_tok * a.out_rows * 4, kBufferDword3);
    for (int b = w; b < (t_hi - t_lo) * TT; b += kGemmWaves) {
      const int tl = b / TT, tt = b - tl * TT;
      const int tok = tt * 16 + (lane >> 2), row = (t_lo + tl) * 16 + 4 * (lane & 3);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(hrs, (lds_void *)(stage + b * 1024), 16,
                                               (tok * a.out_rows + row) * 4, 0, 0, 0);
    }
    if (w == kGemmWaves - 1) {
      const __amdgpu_buffer_rsrc_t grs =
          __builtin_amdgcn_make_buffer_rsrc((void *)a.gain, 0, a.out_rows * 4, kBufferDword3);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(grs, (lds_void *)(stage + kStageGain), 16,
                                               (t_lo * 16 + 4 * lane) * 4, 0, 0, 0);
    }
  }
  // Consumer of RESID_NORM: row t of the sums of squares (kSsGroups floats,
  // 1 KB) into the reduction buffer, reduced after the first pass's loads.
  if (EPI == EPI_SWIGLU && a.ss_in) {
    const __amdgpu_buffer_rsrc_t srs = __builtin_amdgcn_make_buffer_rsrc(
        (void *)a.ss_in, 0, a.n_tok * kSsGroups * 4, kBufferDword3);
    for (int t = w; t < a.n_tok; t += kGemmWaves)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(srs, (lds_void *)((char *)red + t * 1024), 16,
                                               lane * 16, t * 1024, 0, 0);
  }

  for (int gb = t_lo; gb < t_hi; gb += NT) {
    const int n_here = t_hi - gb < NT ? t_hi - gb : NT;
    const int wbytes = n_here * ks * 1024;
    const __amdgpu_buffer_rsrc_t wrs = __builtin_amdgcn_make_buffer_rsrc(
        (void *)((const char *)a.W + (size_t)gb * ks * 1024), 0, wbytes, kBufferDword3);
    int wvo[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) wvo[t] = t < n_here ? t * ks * 1024 + lane * 16 : wbytes;

    i32x4 wr[R][NT], xr[R][TT];
    f32x4 acc[NT][TT];
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int tt = 0; tt < TT; ++tt) acc[t][tt] = f32x4{0.f, 0.f, 0.f, 0.f};
    // loads of this wave's k-step of chunk c (relative to the K range)
    auto issue = [&](int r, int c) {
      const int koff = ((c_begin + c) * 8 + w) * 1024;
#pragma unroll
      for (int tt = 0; tt < TT; ++tt)
        xr[r][tt] = __builtin_amdgcn_raw_buffer_load_b128(xrs, xvo[tt], koff, 0);
#pragma unroll
      for (int t = 0; t < NT; ++t)
        wr[r][t] = __builtin_amdgcn_raw_buffer_load_b128(wrs, wvo[t], koff, kNonTemporal);
    };
    auto mac = [&](int r) {
#pragma unroll
      for (int t = 0; t < NT; ++t)
#pragma unroll
        for (int tt = 0; tt < TT; ++tt)
          acc[t][tt] = mfma16(__builtin_bit_cast(bf16x8, wr[r][t]),
                              __builtin_bit_cast(bf16x8, xr[r][tt]), acc[t][tt]);
    };
    int c = 0;
    if (n_ch >= R) {
      // fill the ring in slot order (the oldest loads are consumed first)
#pragma unroll
      for (int r = 0; r < R; ++r) {
        issue(r, r);
        __builtin_amdgcn_sched_barrier(0);
      }
      // steady state: every consumed slot is refilled R chunks ahead
      for (; c + 2 * R <= n_ch; c += R) {
#pragma unroll
        for (int r = 0; r < R; ++r) {
          mac(r);
          issue(r, c + R + r);
          __builtin_amdgcn_sched_barrier(0);
        }
      }
      // the last one or two rings: refill only while chunks remain
      for (; c < n_ch; c += R) {
#pragma unroll
        for (int r = 0; r < R; ++r) {
          if (c + r < n_ch) {
            mac(r);
            if (c + r + R < n_ch) issue(r, c + r + R);
          }
        }
      }
    } else {
      for (; c < n_ch; ++c) {
        issue(0, c);
        mac(0);
      }
    }

    // Every load of this workgroup has been consumed or is a staging load
    // into LDS: waiting for all of them is free here, and the barriers below
    // make the staged data visible.
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    float *sinv = (float *)stage;  // consumer of RESID_NORM: 1 / rms per token
    if (EPI == EPI_SWIGLU && a.ss_in && gb == t_lo) {
      lds_barrier();
      // 4 threads per token, 64 groups each (16-byte reads staggered by
      // token across the LDS banks; groups past the producer's count are
      // zero), then the 4 quarters in order
      const int t = threadIdx.x >> 2, qtr = threadIdx.x & 3;
      float sum = 0.0f;
      if (t < a.n_tok) {
        const char *row = (const char *)red + t * 1024 + qtr * 256;
#pragma unroll
        for (int j = 0; j < 16; ++j) {
          const f32x4 v = *(const f32x4 *)(row + ((j + t) & 15) * 16);
          sum += (v[0] + v[1]) + (v[2] + v[3]);
        }
      }
      sum += __shfl_xor(sum, 1, 64);
      sum += __shfl_xor(sum, 2, 64);
      if (t < a.n_tok && qtr == 0) sinv[t] = 1.0f / sqrtf(sum / (float)a.norm_dim + a.eps);
      lds_barrier();  // the scales are visible, the reduction buffer is free
    }
    const float2 *rope = rope_lds ? (const float2 *)stage : a.rope;
    const float *sh = (const float *)stage;                  // RESID_NORM residual blocks
    const float *sg = (const float *)(stage + kStageGain);   // RESID_NORM gains
    float *ssq = (float *)(stage + kStageSq);                // RESID_NORM [tile][token]
    // Reduce the 8 waves' partial sums, TPR tiles (all token tiles of each)
    // per LDS round, and run the epilogue on each finished (row pair, token).
#pragma unroll
    for (int t0 = 0; t0 < NT; t0 += TPR) {
      if (t0 < n_here) {
#pragma unroll
        for (int tl = 0; tl < TPR; ++tl)
          if (t0 + tl < NT)
#pragma unroll
            for (int tt = 0; tt < TT; ++tt) red[w][tl * TT + tt][lane] = acc[t0 + tl][tt];
        lds_barrier();
        const int tiles_here = n_here - t0 < TPR ? n_here - t0 : TPR;
        // An item is (accumulator pair, token, g): lanes l1 = token + 16 g and
        // l1 + 32 of the 8 waves' accumulators hold rows 4g .. 4g + 3 and
        // 4g + 8 .. 4g + 11 of the token's column, i.e. the output pairs
        // (p, p + 8) for p = 4g .. 4g + 3.  Items of a 32-lane half-wave
        // share a trip count (items is a multiple of 32).
        const int items = tiles_here * TT * 32;
        for (int it = threadIdx.x; it < items; it += kGemmThreads) {
          const int tok16 = it & 15, g = (it >> 4) & 1, pr = it >> 5;
          const int tl = pr / TT, tt = pr - tl * TT;
          const int tok = tt * 16 + tok16;  // token row
          float sq = 0.0f;
          if (tok < a.n_tok) {
            const int l1 = tok16 + 16 * g;
            f32x4 v1 = red[0][pr][l1], v2 = red[0][pr][l1 + 32];
#pragma unroll
            for (int ww = 1; ww < kGemmWaves; ++ww) {
              v1 += red[ww][pr][l1];
              v2 += red[ww][pr][l1 + 32];
            }
            if constexpr (EPI == EPI_RESID_NORM) {
              sq = resid_norm4(a, sh + (pr * 16 + tok16) * 16, sg + tl * 16, gb + t0 + tl, 4 * g,
                               tok, v1, v2);
            } else {
              if (EPI == EPI_SWIGLU && a.ss_in) {
                const float r = sinv[tok];
                v1 *= r;
                v2 *= r;
              } else if ((EPI == EPI_QKV || EPI == EPI_SWIGLU || EPI == EPI_LOGITS) && a.rs_in) {
                // the RMSNorm scale of the projection's input row
                const float r = a.rs_in[tok];
                v1 *= r;
                v2 *= r;
              }
              epilogue4<EPI>(a, rope, split, gb + t0 + tl, 4 * g, tok, v1, v2);
            }
          }
          if constexpr (EPI == EPI_RESID_NORM) {
            // the two halves (g = 0, 1) of (tile, token): lanes it, it ^ 16
            sq += __shfl_xor(sq, 16, 64);
            if (g == 0) ssq[tl * (TT * 16) + tt * 16 + tok16] = sq;
          }
        }
        lds_barrier();
      }
    }
    if constexpr (EPI == EPI_RESID_NORM) {
      // the group's sum of squares per token, its tiles in order
      if ((int)threadIdx.x < a.n_tok) {
        float sum = 0.0f;
        for (int tl = 0; tl < n_here; ++tl) sum += ssq[tl * (TT * 16) + threadIdx.x];
        a.ss[threadIdx.x * kSsGroups + grp] = sum;
      }
      // group 0 zeroes the row entries of groups that do not exist
      if (grp == 0) {
        const int gap = kSsGroups - a.groups;
        for (int i = threadIdx.x; i < a.n_tok * gap; i += kGemmThreads)
          a.ss[(i / gap) * kSsGroups + a.groups + i % gap] = 0.0f;
      }
      // the last group zeroes the packed columns past the width
      if (grp == a.groups - 1) {
        const int pad = a.xn_ks * 32 - a.out_rows;
        for (int i = threadIdx.x; i < a.n_tok * pad; i += kGemmThreads)
          a.xn[packed_index(i / pad, a.out_rows + i % pad, a.xn_ks)] = 0;
      }
    }
  }
  // LOGITS with fused softmax statistics: the group's logits have been
  // written by its own threads; after the barrier they read them back (from
  // L2, where the stores went) 16 columns at a time: with parts = min(512 /
  // n_tok, the group's tiles), thread i < parts n_tok takes token row
  // i % n_tok and every parts-th tile of the group from tile i / n_tok,
  // leaves its statistics in an LDS slot, and thread t (t < n_tok) combines
  // row t's slots into the group's partial.
  if constexpr (EPI == EPI_LOGITS) {
    if (a.lm_part) {
      __syncthreads();
      LmPart *slot = (LmPart *)(stage + kStageLmSlot);
      const int n_tok = a.n_tok;
      const int V = a.out_rows;
      static_assert(kGemmThreads >= 2 * SB_MAX_ROWS && kGemmThreads * 16 <= kStageBytes,
                    "every token row has a slot of at least two parts in the stage");
      const int nt = t_hi - t_lo;
      const int nl = n_tok > 0 ? n_tok : 1;
      const int parts = kGemmThreads / nl < nt ? kGemmThreads / nl : (nt > 0 ? nt : 1);
      const int t = (int)threadIdx.x % nl, part = (int)threadIdx.x / nl;
      if (n_tok > 0 && part < parts) {
        const __amdgpu_buffer_rsrc_t lrs = __builtin_amdgcn_make_buffer_rsrc(
            (void *)a.logits, 0, n_tok * V * 4, kBufferDword3);
        LmPart r{-INFINITY, INT_MAX, 0.0};
        for (int tile = t_lo + part; tile < t_hi; tile += parts) {
          const int c0 = tile * 16, off = (t * V + c0) * 4;
          float x[16];
          if ((V & 3) == 0) {  // rows 16-byte aligned
#pragma unroll
            for (int j = 0; j < 4; ++j) {
              const f32x4 q = __builtin_bit_cast(
                  f32x4, __builtin_amdgcn_raw_buffer_load_b128(lrs, off + 16 * j, 0, 0));
              x[4 * j] = q[0];
              x[4 * j + 1] = q[1];
              x[4 * j + 2] = q[2];
              x[4 * j + 3] = q[3];
            }
          } else {
#pragma unroll
            for (int j = 0; j < 16; ++j)
              x[j] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(lrs, off + 4 * j, 0, 0));
          }
          lm_merge(r, lm_cols(a, x, c0), a.lm_inv_t, a.lm_greedy);
        }
        slot[part * n_tok + t] = r;
      }
      lds_barrier();
      if ((int)threadIdx.x < n_tok) {
        LmPart r{-INFINITY, INT_MAX, 0.0};
        for (int pp = 0; pp < parts; ++pp) lm_merge(r, slot[pp * n_tok + threadIdx.x], a.lm_inv_t, a.lm_greedy);
        a.lm_part[(size_t)threadIdx.x * a.groups + grp] = r;
      }
    }
  }
  // a workgroup without tiles still owns its staging loads into LDS
  if (t_lo >= t_hi) asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
}


// Wide GEMM (trees of more than 8 token tiles).
//
// A wave owns two 16-row weight tiles (a tile pair) over one of KS parts of
// the workgroup's K range; the 8 / KS pairs of a workgroup (16 / KS tiles)
// share the activation, staged through LDS one chunk at a time: chunk c
// holds k-step c of every K part for all TT token tiles (KS TT fragments of
// 1 KB; the waves load them into registers L chunks ahead, with the
// weights, and write each chunk to one of two LDS buffers when it is due).
// Each fragment read from LDS feeds both tiles of the pair, each weight
// fragment all TT token tiles.  At the end the KS partial sums of each tile
// meet in LDS and the owner wave of the tile runs the epilogue.  Split-K
// launches (the residual projections, whose tile groups are too few to fill
// the chip) also give each of `split` workgroups per tile group a
// contiguous K range; the unit order is K-range-major, so each XCD caches
// one range of the activation.  (Staging by direct-to-LDS loads into
// separate LDS arrays, one per ring buffer, ran the step equally fast; into
// one array the compiler waits for every load in flight before each LDS
// read, since it cannot tell the buffers apart.)
template <int TT, int KS>
struct WideCfg {
  static constexpr int PAIRS = kGemmWaves / KS;                     // tile pairs per workgroup
  static constexpr int FRAG = KS * TT;                              // fragments per chunk
  static constexpr int FPW = (FRAG + kGemmWaves - 1) / kGemmWaves;  // per wave, at most
  static constexpr int FULL = FRAG % kGemmWaves == 0 ? kGemmWaves : FRAG % kGemmWaves;
  static constexpr int L = FRAG <= 18 ? 6 : FRAG <= 36 ? 4 : 2;     // chunks in flight
  static constexpr int LDS = 2 * FRAG > kGemmWaves * TT ? 2 * FRAG : kGemmWaves * TT;  // KB
  static_assert(L % 2 == 0, "the unrolled chunk steps cover both LDS buffers");
  static_assert((L - 1) * (FPW + 2) <= 63, "the loads in flight fit the wait counter");
  static_assert(LDS <= 160, "the chunk buffers and the reduction fit LDS");
};

template <int EPI, int TT, int KS>
__global__ __launch_bounds__(kGemmThreads, 1) void k_gemm_wide(GemmArgs a) {
  using C = WideCfg<TT, KS>;
  constexpr int L = C::L, FPW = C::FPW;
  constexpr int NW = 2;  // weight loads per wave per chunk (one per tile)
  __shared__ __attribute__((aligned(16))) char abuf[C::LDS * 1024];
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int ks = a.ks;
  const int nb = gridDim.x;
  const int u = (nb & 7) == 0 ? (blockIdx.x & 7) * (nb >> 3) + (blockIdx.x >> 3) : blockIdx.x;
  const int split = u / a.groups, grp = u - split * a.groups;
  const int pw = w % C::PAIRS, kp = w / C::PAIRS;  // tile pair, K part
  const int tile0 = (grp * C::PAIRS + pw) * 2;
  const bool has = tile0 < a.tiles;  // wave-uniform
  // K part q of the Q = split KS parts of the launch: k-steps [kb(q), kb(q+1))
  const int Q = a.split * KS;
  auto kb = [&](int q) { return ks * q / Q; };
  const int nchunk = (ks + Q - 1) / Q;  // chunks: one k-step of every part
  const int xbytes = ((a.n_tok + 15) >> 4) * ks * 1024;
  const __amdgpu_buffer_rsrc_t xrs =
      __builtin_amdgcn_make_buffer_rsrc((void *)a.X, 0, xbytes, kBufferDword3);
  const int wbytes = a.tiles * ks * 1024;
  const __amdgpu_buffer_rsrc_t wrs =
      __builtin_amdgcn_make_buffer_rsrc((void *)a.W, 0, wbytes, kBufferDword3);
  const int qw = split * KS + kp;  // this wave's K part
  const int kw0 = kb(qw), kwn = kb(qw + 1) - kw0;
  int wvo[NW];
#pragma unroll
  for (int j = 0; j < NW; ++j)
    wvo[j] = tile0 + j < a.tiles ? (tile0 + j) * ks * 1024 + lane * 16 : wbytes;
  // waves w < FULL move FPW fragments per chunk, the others FPW - 1
  const bool full = w < C::FULL;

  // Chunk c's fragment f = p TT + tt (K part p, token tile tt) sits at KB f
  // of its buffer; wave w moves fragments w + 8 j.  Lane l loads bytes
  // 16 l .. of a fragment (token row r = l / 4, k 8 (l % 4) ..) and stores
  // them at 16-byte slot 4 r + ((l % 4) ^ x(r)), x(r) = (r / 2 ^ r / 8) % 4:
  // the 8 (16) lanes that a 128-bit LDS access serves per clock then cover
  // all 32 (64) banks, for the writes and for the operand reads.
  auto xsw = [](int r) { return ((r >> 1) ^ (r >> 3)) & 3; };
  const int wsw = ((lane >> 2) * 4 + ((lane & 3) ^ xsw(lane >> 2))) * 16;
  const int rsw = ((lane & 15) * 4 + ((lane >> 4) ^ xsw(lane & 15))) * 16;
  // per fragment of this wave: its lane offset at k-step 0 of its K part
  // and the part's length (the loop below only adds the chunk)
  int xoff[FPW], xlen[FPW];
#pragma unroll
  for (int j = 0; j < FPW; ++j) {
    const int f = w + kGemmWaves * j;
    const int p = f / TT, tt = f - p * TT;
    const int q = split * KS + p;
    const int k0 = kb(q);
    xoff[j] = (tt * ks + k0) * 1024 + lane * 16;
    xlen[j] = kb(q + 1) - k0;
  }
  i32x4 xr[L][FPW], wr[L][NW];
  auto issue = [&](int c, int slot) {
#pragma unroll
    for (int j = 0; j < FPW; ++j)
      if (j < FPW - 1 || full)
        xr[slot][j] = __builtin_amdgcn_raw_buffer_load_b128(
            xrs, c < xlen[j] ? xoff[j] + c * 1024 : xbytes, 0, 0);
    const bool in = c < kwn;
#pragma unroll
    for (int j = 0; j < NW; ++j)
      wr[slot][j] = __builtin_amdgcn_raw_buffer_load_b128(wrs, in ? wvo[j] : wbytes,
                                                          (kw0 + (in ? c : 0)) * 1024, kNonTemporal);
  };
  auto stage = [&](int slot, int buf) {
#pragma unroll
    for (int j = 0; j < FPW; ++j)
      if (j < FPW - 1 || full)
        *(i32x4 *)(abuf + (buf * C::FRAG + w + kGemmWaves * j) * 1024 + wsw) = xr[slot][j];
  };
  f32x4 acc[NW][TT];
#pragma unroll
  for (int j = 0; j < NW; ++j)
#pragma unroll
    for (int tt = 0; tt < TT; ++tt) acc[j][tt] = f32x4{0.f, 0.f, 0.f, 0.f};
  auto mac = [&](int buf, int slot) {
#pragma unroll
    for (int tt = 0; tt < TT; ++tt) {
      // operand B: token row lane % 16, k 8 (lane / 16) .. of the fragment
      const uint4 xv = *(const uint4 *)(abuf + (buf * C::FRAG + kp * TT + tt) * 1024 + rsw);
#pragma unroll
      for (int j = 0; j < NW; ++j)
        acc[j][tt] = mfma16(__builtin_bit_cast(bf16x8, wr[slot][j]), as_bf16x8(xv), acc[j][tt]);
    }
  };
  // One group of loads per chunk (its activation, then its weights), L
  // groups ahead.  Step c writes chunk c + 1's activation to LDS while it
  // multiplies chunk c, then one barrier: chunk c + 1 is visible for the
  // next step and every wave is done with buffer c % 2, which the next step
  // overwrites.  At step c the loads issued after chunk c + 1's group are
  // L - 2 whole groups.
  constexpr int AFTER_FULL = (L - 2) * (FPW + NW), AFTER_SHORT = (L - 2) * (FPW - 1 + NW);
  auto wait_next = [&]() {
    if (full)
      asm volatile("s_waitcnt vmcnt(%0)" ::"n"(AFTER_FULL + FPW + NW) : "memory");
    else
      asm volatile("s_waitcnt vmcnt(%0)" ::"n"(AFTER_SHORT + FPW - 1 + NW) : "memory");
  };
#pragma unroll
  for (int c = 0; c < L; ++c) issue(c, c);
  wait_next();  // chunk 0
  stage(0, 0);
  lds_barrier();
  __builtin_amdgcn_sched_barrier(0);
  for (int c0 = 0; c0 < nchunk; c0 += L) {
#pragma unroll
    for (int i = 0; i < L; ++i) {
      const int c = c0 + i;
      if (c >= nchunk) break;  // uniform
      if (full)
        asm volatile("s_waitcnt vmcnt(%0)" ::"n"(AFTER_FULL) : "memory");
      else
        asm volatile("s_waitcnt vmcnt(%0)" ::"n"(AFTER_SHORT) : "memory");
      stage((i + 1) % L, (i + 1) % 2);
      if (has) mac(i % 2, i);
      lds_barrier();
      __builtin_amdgcn_sched_barrier(0);
      issue(c + L, i);
    }
  }
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  // Reduction, one tile of the pairs per round: every wave leaves its
  // partial sums of the pair's tile j in LDS; the wave of K part j adds the
  // KS partials of its pair in part order and runs the epilogue.
  f32x4(*red)[64] = (f32x4(*)[64])abuf;  // [wave][tt][lane]
#pragma unroll
  for (int j = 0; j < NW; ++j) {
    lds_barrier();
#pragma unroll
    for (int tt = 0; tt < TT; ++tt) red[w * TT + tt][lane] = acc[j][tt];
    lds_barrier();
    const int tile = tile0 + j;
    if (kp == j && tile < a.tiles) {
#pragma unroll 1
      for (int tt = 0; tt < TT; ++tt) {
        f32x4 v = red[pw * TT + tt][lane];
#pragma unroll
        for (int p = 1; p < KS; ++p) v += red[(p * C::PAIRS + pw) * TT + tt][lane];
        // lane l holds rows 4 (l / 16) .. + 3 of the tile for token row
        // l % 16; lanes l < 32 take rows p0 = 4 (l / 16) .. + 3 and
        // p0 + 8 .. + 3 (from lane l + 32)
        f32x4 v2;
#pragma unroll
        for (int i = 0; i < 4; ++i) v2[i] = __shfl_down(v[i], 32, 64);
        const int tok = tt * 16 + (lane & 15);
        if (lane < 32 && tok < a.n_tok) {
          if ((EPI == EPI_QKV || EPI == EPI_SWIGLU || EPI == EPI_LOGITS) && a.rs_in) {
            const float r = a.rs_in[tok];
            v *= r;
            v2 *= r;
          }
          epilogue4<EPI>(a, a.rope, split, tile, 4 * (lane >> 4), tok, v, v2);
        }
      }
    }
  }
}

template <int EPI, int TT, int KS>
hipError_t launch_wide_tt(const GemmArgs &a, int grid, hipStream_t s) {
  LaunchEvents &ev = g_launch_events;
  if (!ev.taken) {
    ev.taken = true;
    hipExtLaunchKernelGGL((k_gemm_wide<EPI, TT, KS>), dim3(grid), dim3(kGemmThreads), 0, s,
                          ev.start, ev.stop, 0, a);
  } else {
    hipLaunchKernelGGL((k_gemm_wide<EPI, TT, KS>), dim3(grid), dim3(kGemmThreads), 0, s, a);
  }
  return hipGetLastError();
}

template <int EPI, int KS>
hipError_t launch_wide_ks(const GemmArgs &a, int tt, int grid, hipStream_t s) {
  switch (tt) {
    case 9: return launch_wide_tt<EPI, 9, KS>(a, grid, s);
    case 12: return launch_wide_tt<EPI, 12, KS>(a, grid, s);
    case 16: return launch_wide_tt<EPI, 16, KS>(a, grid, s);
    default: return hipErrorInvalidValue;
  }
}

template <int EPI, int TT, int NT>
hipError_t launch_tt_nt(const GemmArgs &a, int grid, hipStream_t s) {
  if constexpr (NT > gemm_nt_cap(TT)) {
    return hipErrorInvalidValue;
  } else {
    LaunchEvents &ev = g_launch_events;
    if (!ev.taken) {
      ev.taken = true;
      hipExtLaunchKernelGGL((k_gemm<EPI, TT, NT>), dim3(grid), dim3(kGemmThreads), 0, s, ev.start,
                            ev.stop, 0, a);
    } else {
      hipLaunchKernelGGL((k_gemm<EPI, TT, NT>), dim3(grid), dim3(kGemmThreads), 0, s, a);
    }
    return hipGetLastError();
  }
}

template <int EPI, int TT>
hipError_t launch_tt(const GemmArgs &a, int nt, int grid, hipStream_t s) {
  switch (nt) {
    case 1: return launch_tt_nt<EPI, TT, 1>(a, grid, s);
    case 2: return launch_tt_nt<EPI, TT, 2>(a, grid, s);
    case 3: return launch_tt_nt<EPI, TT, 3>(a, grid, s);
    case 4: return launch_tt_nt<EPI, TT, 4>(a, grid, s);
    case 6: return launch_tt_nt<EPI, TT, 6>(a, grid, s);
    case 8: return launch_tt_nt<EPI, TT, 8>(a, grid, s);
    default: return hipErrorInvalidValue;
  }
}

// Launch of a planned GEMM with epilogue EPI (the kernel for its token
// tiles and tiles per pass).
template <int EPI>
hipError_t launch_epi(const GemmArgs &b, const GemmPlan &p, hipStream_t s) {
  if constexpr (EPI == EPI_SWIGLU || EPI == EPI_RESID || EPI == EPI_LOGITS) {
    if (p.wide == 2) return launch_wide_ks<EPI, 2>(b, p.tt, p.grid, s);
  }
  if constexpr (EPI == EPI_QKV || EPI == EPI_RESID) {
    if (p.wide == 4) return launch_wide_ks<EPI, 4>(b, p.tt, p.grid, s);
  }
  if (p.wide) return hipErrorInvalidValue;
  switch (p.tt) {
    case 1: return launch_tt<EPI, 1>(b, p.nt, p.grid, s);
    case 2: return launch_tt<EPI, 2>(b, p.nt, p.grid, s);
    case 3: return launch_tt<EPI, 3>(b, p.nt, p.grid, s);
    case 4: return launch_tt<EPI, 4>(b, p.nt, p.grid, s);
    case 5: return launch_tt<EPI, 5>(b, p.nt, p.grid, s);
    case 6: return launch_tt<EPI, 6>(b, p.nt, p.grid, s);
    case 8: return launch_tt<EPI, 8>(b, p.nt, p.grid, s);
    case 12: return launch_tt<EPI, 12>(b, p.nt, p.grid, s);
    case 16: return launch_tt<EPI, 16>(b, p.nt, p.grid, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace
}  // namespace sb
