// Skinny matrix-core GEMM with fused epilogues (RoPE + KV write, residual
// delta, SwiGLU, logits) for gfx950.
//
// The verify forward multiplies n_rows (5..256) activation rows by every
// weight matrix once; the weights (13-140 GB) dominate the bytes, so the
// GEMM streams each weight tile from HBM exactly once with 16-byte loads in
// the operand order of v_mfma_f32_16x16x32_bf16 (the layout sb_pack_weight
// writes).  One workgroup per compute unit owns a range of weight tiles and
// walks K in chunks, reusing each activation fragment across all of its
// tiles; the residual projections, about one tile per compute unit, also
// split K across workgroups and leave partial deltas for the next RMSNorm.
#include <math.h>

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

// Epilogue of one finished output pair: rows p and p + 8 of tile `tile`,
// activation row t < n_tok, values v1 / v2 (K range `split` of a split-K
// launch).
__device__ __forceinline__ void epilogue(const GemmArgs &a, const float2 *rope, int split,
                                         int tile, int p, int t, float v1, float v2) {
  if (a.epi == EPI_QKV) {
    const int d = a.head_dim, ht = d / 16;
    const int qt = a.n_heads * ht, kt = a.n_kv * ht;
    if (tile < qt + kt) {
      const bool isq = tile < qt;
      const int idx = isq ? tile : tile - qt;
      const int head = idx / ht, u = idx % ht;
      const int j = 8 * u + p;
      float o1, o2;
      rope_pair(v1, v2, rope[t * (d / 2) + j], &o1, &o2);
      uint16_t *dst = isq ? a.q + ((size_t)t * a.n_heads + head) * d
                          : a.kc + ((size_t)head * a.cap + a.kv_len + t) * d;
      dst[j] = f2bf(o1);
      dst[j + d / 2] = f2bf(o2);
    } else {
      // V is cached transposed: [head][d][slot]
      const int idx = tile - qt - kt;
      const int head = idx / ht, u = idx % ht;
      uint16_t *col = a.vc + ((size_t)head * d + 16 * u + p) * a.cap + a.kv_len + t;
      col[0] = f2bf(v1);
      col[(size_t)8 * a.cap] = f2bf(v2);
    }
  } else if (a.epi == EPI_RESID) {
    // the projection is stored as a delta (one slice per K range); the next
    // RMSNorm adds the slices to the residual stream
    const int d1 = tile * 16 + p, d2 = d1 + 8;
    float *drow = a.h + ((size_t)split * a.n_tok + t) * a.out_rows;
    if (d1 < a.out_rows) drow[d1] = v1;
    if (d2 < a.out_rows) drow[d2] = v2;
  } else if (a.epi == EPI_SWIGLU) {
    const int f = tile * 8 + p;
    const float gsil = v1 / (1.0f + expf(-v1));
    a.act[packed_index(t, f, a.act_ks)] = f2bf(gsil * v2);
  } else {  // EPI_LOGITS
    const int v1i = tile * 16 + p, v2i = v1i + 8;
    float *lrow = a.logits + (size_t)t * a.out_rows;
    if (v1i < a.out_rows) lrow[v1i] = v1;
    if (v2i < a.out_rows) lrow[v2i] = v2;
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
// about 48 for the rest).
template <int TT, int NT>
struct Ring {
  static constexpr int free_regs = 208 - TT - NT - 4 * NT * TT;
  static constexpr int r = free_regs / (4 * (NT + TT));
  static constexpr int R = r > 4 ? 4 : (r < 1 ? 1 : r);
};

// (tile, token tile) accumulator pairs reduced per LDS round (128 KB)
constexpr int kRedPairs = 16;
// RoPE table staged in LDS for the QKV epilogue (float2 entries)
constexpr int kRopeLds = 4096;

// Workgroup barrier for LDS traffic only (does not wait for global loads).
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

template <int TT, int NT>
__global__ __launch_bounds__(kGemmThreads, 1) void k_gemm(GemmArgs a) {
  __shared__ f32x4 red[kGemmWaves][kRedPairs][64];
  __shared__ float2 srope[kRopeLds];
  constexpr int R = Ring<TT, NT>::R;
  constexpr int TPR = kRedPairs / TT > 0 ? kRedPairs / TT : 1;  // tiles per reduction round
  // wave-uniform quantities live in scalar registers
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int ks = a.ks;
  const int S = a.split;
  const int split = blockIdx.x % S, grp = blockIdx.x / S;
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
    xvo[tt] = (tt * 16 + (lane & 15)) < a.n_tok ? tt * ks * 1024 + lane * 16 : xbytes;

  // QKV: the step's RoPE table goes to LDS by direct-to-LDS loads issued
  // now (no registers held; each wave instruction moves 1 KB), ready long
  // before the epilogue.  The table buffer holds whole 1 KB blocks
  // (rows padded to 16).
  const bool rope_lds = a.epi == EPI_QKV && a.n_tok * (a.head_dim / 2) <= kRopeLds;
  if (rope_lds) {
    const int nblk = (a.n_tok * (a.head_dim / 2) * 8 + 1023) >> 10;
    for (int b = w; b < nblk; b += kGemmWaves)
      __builtin_amdgcn_global_load_lds((const void *)((const char *)a.rope + b * 1024 + lane * 16),
                                       (__attribute__((address_space(3))) void *)((char *)srope + b * 1024),
                                       16, 0, 0);
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

    // Reduce the 8 waves' partial sums, TPR tiles (all token tiles of each)
    // per LDS round, and run the epilogue on each finished (row pair, token).
    // Every load of this workgroup has been consumed (or is a RoPE load to
    // LDS): waiting for all of them here is free and makes the staged table
    // visible after the barrier.
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    const float2 *rope = rope_lds ? srope : a.rope;
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
        const int items = tiles_here * TT * 128;
        for (int it = threadIdx.x; it < items; it += kGemmThreads) {
          const int p = it & 7;
          const int rest = it >> 3;
          const int tl = rest / (TT * 16);
          const int tok = rest - tl * (TT * 16);
          const int tt = tok >> 4;
          if (tok < a.n_tok) {
            const int l1 = (tok & 15) + 16 * (p >> 2), e1 = p & 3;
            const int l2 = (tok & 15) + 16 * ((p + 8) >> 2), e2 = (p + 8) & 3;
            float v1 = 0.f, v2 = 0.f;
#pragma unroll
            for (int ww = 0; ww < kGemmWaves; ++ww) {
              v1 += red[ww][tl * TT + tt][l1][e1];
              v2 += red[ww][tl * TT + tt][l2][e2];
            }
            epilogue(a, rope, split, gb + t0 + tl, p, tok, v1, v2);
          }
        }
        lds_barrier();
      }
    }
  }
  // a workgroup without tiles still owns its RoPE loads into LDS
  if (rope_lds) asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
}

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

// Token-tile counts with a kernel (rounded up; padded rows read as zero) and
// the largest tile count per pass each supports.
constexpr int kTTs[] = {1, 2, 3, 4, 6, 8, 12, 16};
constexpr int kNTs[] = {1, 2, 3, 4, 6, 8};
constexpr int nt_cap(int tt) { return tt <= 4 ? 8 : tt <= 6 ? 6 : tt <= 8 ? 4 : tt <= 12 ? 2 : 1; }

template <int TT, int NT>
hipError_t launch_tt_nt(const GemmArgs &a, int grid, hipStream_t s) {
  if constexpr (NT > nt_cap(TT)) {
    return hipErrorInvalidValue;
  } else {
    hipLaunchKernelGGL((k_gemm<TT, NT>), dim3(grid), dim3(kGemmThreads), 0, s, a);
    return hipGetLastError();
  }
}

template <int TT>
hipError_t launch_tt(const GemmArgs &a, int nt, int grid, hipStream_t s) {
  switch (nt) {
    case 1: return launch_tt_nt<TT, 1>(a, grid, s);
    case 2: return launch_tt_nt<TT, 2>(a, grid, s);
    case 3: return launch_tt_nt<TT, 3>(a, grid, s);
    case 4: return launch_tt_nt<TT, 4>(a, grid, s);
    case 6: return launch_tt_nt<TT, 6>(a, grid, s);
    case 8: return launch_tt_nt<TT, 8>(a, grid, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

GemmPlan plan_gemm(int epi, int tiles, int ks, int n_tok) {
  GemmPlan p{};
  const int cus = device_cus();
  const int nc = ks / 8;
  const int tt = (n_tok + 15) / 16;
  for (int v : kTTs)
    if (v >= tt) {
      p.tt = v;
      break;
    }
  // Projections that add into the residual stream have as many tiles as the
  // model is wide, about one per compute unit: they split K so that each
  // workgroup owns several tiles; the next RMSNorm sums the partial deltas.
  const int per_cu = (tiles + cus - 1) / cus;
  int S = 1;
  if (epi == EPI_RESID) S = per_cu == 1 ? kMaxSplit : per_cu == 2 ? 2 : 1;
  if (S > nc) S = nc;
  if (S < 1) S = 1;
  int groups = cus / S;
  if (groups > tiles) groups = tiles;
  const int per_wg = (tiles + groups - 1) / groups;
  const int cap = nt_cap(p.tt);
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

hipError_t launch_gemm(int epi, const GemmArgs &a, int tiles, int *split, hipStream_t s) {
  if (a.ks % 8 != 0 || a.n_tok <= 0 || a.n_tok > SB_MAX_ROWS) return hipErrorInvalidValue;
  const GemmPlan p = plan_gemm(epi, tiles, a.ks, a.n_tok);
  GemmArgs b = a;
  b.epi = epi;
  b.tiles = tiles;
  b.split = p.split;
  b.groups = p.groups;
  if (split) *split = p.split;
  switch (p.tt) {
    case 1: return launch_tt<1>(b, p.nt, p.grid, s);
    case 2: return launch_tt<2>(b, p.nt, p.grid, s);
    case 3: return launch_tt<3>(b, p.nt, p.grid, s);
    case 4: return launch_tt<4>(b, p.nt, p.grid, s);
    case 6: return launch_tt<6>(b, p.nt, p.grid, s);
    case 8: return launch_tt<8>(b, p.nt, p.grid, s);
    case 12: return launch_tt<12>(b, p.nt, p.grid, s);
    case 16: return launch_tt<16>(b, p.nt, p.grid, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace sb
