// Persistent verify forward of a bf16 decoder (gfx950): every layer of the
// target forward in one cooperative launch.
//
// The step is bound by HBM: its bytes are the weights (read once) and the
// prefix KV.  Run as a chain of kernels, every GEMM and attention launch
// pays a ramp (dispatch, first-load latency) and a tail during which the
// memory system idles; a layer has seven such boundaries.  Here one
// workgroup of 512 threads runs on every compute unit for the whole
// forward, and the phases of a layer
//
//   QKV GEMM (+ 1/rms, RoPE, K/V write) | attention (key ranges) |
//   range merge | O GEMM (split-K slices) | residual add + RMSNorm partials |
//   gate/up GEMM (+ 1/rms, SwiGLU) | down GEMM (split-K slices) |
//   residual add + RMSNorm partials of the next layer's input
//
// are separated by device-wide barriers.  Weights do not depend on the
// previous phase, so before each barrier the workgroup requests the first
// chunks of its next GEMM's weights into LDS (and the attention phase its
// prefix K rows into registers): the barrier overlaps with weight streaming.
//
// Measured on MI355X (7B shape, 33 rows): 4.40 ms per forward against
// 3.44 ms for the chain of kernels.  A device-wide barrier costs 1.2-4 us
// from the last arrival to the first departure -- about what a kernel launch
// costs -- and the 64 KB per compute unit that can be prefetched covers
// about 2 us of it; the GEMM phases run no faster than the standalone GEMM
// kernels.  The chain is the default (SB_FWD_AUTO); this kernel is the
// SB_FWD_PERSISTENT form, one launch per forward.
//
// Data handed from one workgroup to another inside the kernel is stored with
// device-scope (sc1) stores, which write through the XCD's L2, and read with
// device-scope loads, which do not hit a stale line in the reader's L2; the
// barrier waits for the stores to complete before it arrives.  Weights and
// the committed prefix KV are never written here and are read with ordinary
// (non-temporal) loads.
//
// The barrier: every workgroup adds 1 to the counter of its group of
// workgroups (blockIdx mod 8), one wave polls the 8 counters until each
// reaches its target, with a time limit (a barrier that does not complete
// sets the status word, and every later barrier fails at once, so the
// kernel always ends).  A cooperative launch guarantees that every
// workgroup is resident.
#pragma once

#include <math.h>

#include "sb_gemm_kernel.h"

namespace sb {
namespace {

constexpr int kPkThreads = kPkThreadsHost;
constexpr int kPkWaves = kPkThreads / 64;
constexpr int kDev = 16;  // cache policy bit sc1: device-scope access
// LDS: the GEMM's reduction buffer (128 KB) then its staging area (32 KB);
// the attention phase reuses the same bytes.
constexpr int kRedBytes = kGemmWaves * kRedPairs * 64 * 16;
constexpr int kPkLds = kRedBytes + kStageBytes;
// The last 512 bytes of the LDS block: the barrier's flag (at -512) and the
// tokens' RMSNorm scales 1/rms (64 floats at -256); nothing else reaches
// them (the RoPE table is staged only when it leaves them free).
constexpr int kPkOkOff = kPkLds - 512;
constexpr int kPkInvOff = kPkLds - 256;
// barrier time limit, in ticks of the 100 MHz s_memrealtime counter (2 s)
constexpr unsigned long long kPkSpinTicks = 200000000ull;

// Thread and workgroup index, read through an empty asm so that values
// derived from them are computed where a phase uses them: without it the
// compiler hoists every phase's lane offsets out of the layer loop and
// keeps all of them live across the whole forward.
__device__ __forceinline__ int tid() {
  int t = threadIdx.x;
  asm volatile("" : "+v"(t));
  return t;
}
__device__ __forceinline__ int vopaque(int v) {
  asm volatile("" : "+v"(v));
  return v;
}
__device__ __forceinline__ int sopaque(int v) {
  asm volatile("" : "+s"(v));
  return v;
}
__device__ __forceinline__ int bid() {
  int b = blockIdx.x;
  asm volatile("" : "+s"(b));
  return b;
}

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const void *p, long long bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(uniform_ptr(p), 0,
                                           __builtin_amdgcn_readfirstlane((int)bytes), kBufferDword3);
}

__device__ __forceinline__ void s_barrier_only() {
  asm volatile("s_barrier" ::: "memory");
}

// ---------------------------------------------------------------------------
// device-wide barrier
// ---------------------------------------------------------------------------

// Completes this workgroup's stores (every wave waits for its own), then the
// caller may issue prefetch loads in waves 1..7 before pk_wait.
__device__ __forceinline__ void pk_drain() {
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  s_barrier_only();
}

// Wave 0 arrives and polls; every wave leaves when all workgroups have
// arrived.  Returns false (for the whole workgroup) when the time limit
// passed or an earlier barrier failed.  bi: this workgroup's barrier count.
__device__ __forceinline__ bool pk_wait(PkSync *sy, unsigned &bi, int *s_ok) {
  const int nb = gridDim.x;
  if (tid() == 0) {
    int ok = 1;
    __hip_atomic_fetch_add(&sy->grp[bid() & 7][0], 1u, __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
    const unsigned long long t0 = __builtin_amdgcn_s_memrealtime();
    for (;;) {
      bool done = true;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const unsigned n = (unsigned)((nb - j + 7) >> 3);
        done &= __hip_atomic_load(&sy->grp[j][0], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) >=
                (bi + 1) * n;
      }
      if (done) break;
      if (__hip_atomic_load(&sy->status[0], __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) != 0 ||
          __builtin_amdgcn_s_memrealtime() - t0 > kPkSpinTicks) {
        __hip_atomic_fetch_or(&sy->status[0], 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        ok = 0;
        break;
      }
      __builtin_amdgcn_s_sleep(1);
    }
    *s_ok = ok;
  }
  ++bi;
  // the flag is in LDS: wait for wave 0's LDS write, then everybody reads it
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  s_barrier_only();
  return *(volatile int *)s_ok != 0;
}

// ---------------------------------------------------------------------------
// GEMM phase
// ---------------------------------------------------------------------------

// LDS map of a GEMM stage (offsets in the 160 KB block):
//   [0, kPfBytes)              the pass's first chunks of weights, loaded by
//                              direct-to-LDS loads (for the first pass before
//                              the stage's barrier), free once consumed;
//   [kSsOff, kRedBytes)        the tokens' rows of RMSNorm partial sums (in
//                              run), pk_norm's row partials (in a light phase);
//   [0, kRedBytes)             the waves' partial sums, after the main loop;
//   [kRedBytes, + kStageBytes) the RoPE table; the flag and 1/rms at its end.
constexpr int kPfBytes = 64 * 1024;
constexpr int kSsOff = kPfBytes;

struct GemmIO {
  const uint16_t *W;  // packed weights
  const uint16_t *X;  // packed activations (written in this kernel)
  int scale_rows;     // consumers of an RMSNorm: 1/rms from the ss partials
  // QKV
  uint16_t *kc, *vc;  // this layer's caches
  // RESID: delta slices; LOGITS: logits; SWIGLU: act
  float *out_f;
  uint16_t *out_b;
  int out_ks;
};

// The LDS offset `off`, usable once the wave's load into x has completed:
// memory loads complete in issue order, so every load the wave issued
// before x's -- the direct-to-LDS weight loads among them -- has landed.
__device__ __forceinline__ int lds_after(int off, const i32x4 &x) {
  asm volatile("" : "+v"(off) : "v"(x[0]));
  return off;
}

template <int EPI, int TT, int NT>
struct PkGemm {
  static constexpr int R = Ring<TT, NT>::R;
  // chunks of each pass whose weights come through LDS
  static constexpr int PF0 = kPfBytes / (NT * kPkWaves * 1024);
  static constexpr int P = PF0 < R ? PF0 : R;
  static constexpr int TPR = kRedPairs / TT > 0 ? kRedPairs / TT : 1;
  PkGemmPlan p;
  int t_lo, t_hi, split, grp, c_begin, n_ch;

  __device__ __forceinline__ void plan(const PkGemmPlan &pl) {
    p = pl;
    const int nb = gridDim.x, b = bid();
    // work unit u = (tile group, K range), numbered XCD-major (workgroup b
    // runs on XCD b mod 8): each XCD streams one contiguous part of W
    const int u = (nb & 7) == 0 ? (b & 7) * (nb >> 3) + (b >> 3) : b;
    const int units = p.split * p.groups;
    split = u % p.split;
    grp = u / p.split;
    if (u < units) {
      t_lo = (int)(((long long)p.tiles * grp) / p.groups);
      t_hi = (int)(((long long)p.tiles * (grp + 1)) / p.groups);
    } else {
      t_lo = t_hi = 0;
    }
    const int nc = p.ks >> 3;
    c_begin = (nc * split) / p.split;
    n_ch = (nc * (split + 1)) / p.split - c_begin;
  }

  // Direct-to-LDS loads of this wave's k-step of chunks 0 .. P-1 of the
  // pass starting at tile gb: 1 KB per (chunk, tile) at
  // ((chunk * NT + tile) * 8 + wave) KB; tiles past the group read zero.
  __device__ __forceinline__ void prefetch(const uint16_t *W, int gb, char *smem) {
    if (gb >= t_hi) return;
    const int w = __builtin_amdgcn_readfirstlane(tid() >> 6);
    const int lane = tid() & 63;
    const int n_here = t_hi - gb < NT ? t_hi - gb : NT;
    const int wbytes = n_here * p.ks * 1024;
    const __amdgpu_buffer_rsrc_t rs = rsrc((const char *)W + (size_t)gb * p.ks * 1024, wbytes);
#pragma unroll
    for (int pp = 0; pp < P; ++pp) {
      if (pp < n_ch) {
        const int koff = ((c_begin + pp) * 8 + w) * 1024;
#pragma unroll
        for (int t = 0; t < NT; ++t)
          __builtin_amdgcn_raw_ptr_buffer_load_lds(
              rs, (lds_void *)(smem + ((pp * NT + t) * kPkWaves + w) * 1024), 16,
              t < n_here ? t * p.ks * 1024 + lane * 16 : wbytes, koff, 0, kNonTemporal);
      }
    }
  }

  // prefetched: waves 1..7 issued the first pass's prefetch before the
  // stage's barrier (wave 0, which polled it, issues its own here).
  __device__ __forceinline__ void run(const PkArgs &a, const GemmIO &io, char *smem, bool prefetched) {
    f32x4(*red)[kRedPairs][64] = (f32x4(*)[kRedPairs][64])smem;
    char *stage = smem + kRedBytes;
    const int w = __builtin_amdgcn_readfirstlane(tid() >> 6);
    const int lane = tid() & 63;
    const int ks = p.ks;
    const int n_tok = a.n_tok;
    const int nwg = gridDim.x;
    if (!prefetched || w == 0) prefetch(io.W, t_lo, smem);

    // staging into LDS by direct-to-LDS loads: the step's RoPE table (QKV),
    // and each token's row of RMSNorm partial sums (consumers of a norm)
    const bool rope_lds = EPI == EPI_QKV && n_tok * (a.head_dim / 2) * 8 <= kStageBytes - 512;
    if (rope_lds) {
      const int nblk = (n_tok * (a.head_dim / 2) * 8 + 1023) >> 10;
      for (int b = w; b < nblk; b += kPkWaves)
        __builtin_amdgcn_global_load_lds((const void *)((const char *)a.rope + b * 1024 + lane * 16),
                                         (lds_void *)(stage + b * 1024), 16, 0, 0);
    }
    if (io.scale_rows && t_lo < t_hi) {
      const __amdgpu_buffer_rsrc_t srs = rsrc(a.ss, (long long)n_tok * kSsGroups * 4);
      for (int t = w; t < n_tok; t += kPkWaves)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(srs, (lds_void *)(smem + kSsOff + t * 1024), 16,
                                                 lane * 16, t * 1024, 0, kDev);
    }

    const int xbytes = ((n_tok + 15) >> 4) * ks * 1024;
    const __amdgpu_buffer_rsrc_t xrs = rsrc(io.X, xbytes);
    int xvo[TT];
#pragma unroll
    for (int tt = 0; tt < TT; ++tt)
      xvo[tt] = (tt * 16 + (lane & 15)) < n_tok
                    ? tt * ks * 1024 + (lane & 15) * 64 + (lane >> 4) * 16
                    : xbytes;

    for (int gb = t_lo; gb < t_hi; gb += NT) {
      const int n_here = t_hi - gb < NT ? t_hi - gb : NT;
      if (gb != t_lo) prefetch(io.W, gb, smem);  // LDS is free again after the last epilogue
      const int wbytes = n_here * ks * 1024;
      const __amdgpu_buffer_rsrc_t wrs = rsrc((const char *)io.W + (size_t)gb * ks * 1024, wbytes);
      int wvo[NT];
#pragma unroll
      for (int t = 0; t < NT; ++t) wvo[t] = t < n_here ? t * ks * 1024 + lane * 16 : wbytes;
      i32x4 wr[R][NT], xr[R][TT];
      f32x4 acc[NT][TT];
#pragma unroll
      for (int t = 0; t < NT; ++t)
#pragma unroll
        for (int tt = 0; tt < TT; ++tt) acc[t][tt] = f32x4{0.f, 0.f, 0.f, 0.f};
      auto issue_x = [&](int r, int c) {
        const int koff = ((c_begin + c) * 8 + w) * 1024;
#pragma unroll
        for (int tt = 0; tt < TT; ++tt)
          xr[r][tt] = __builtin_amdgcn_raw_buffer_load_b128(xrs, xvo[tt], koff, kDev);
      };
      auto issue_w = [&](int r, int c) {
        const int koff = ((c_begin + c) * 8 + w) * 1024;
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
      // fill: the register weights of chunks P .. R-1, then the activations
      // of chunks 0 .. R-1 (issued after every prefetch of this wave)
#pragma unroll
      for (int r = P; r < R; ++r)
        if (r < n_ch) issue_w(r, r);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int r = 0; r < R; ++r)
        if (r < n_ch) issue_x(r, r);
      __builtin_amdgcn_sched_barrier(0);
      // the first ring: chunks 0 .. P-1 take their weights from LDS
      const int lbase = lds_after(w * 1024 + lane * 16, xr[0][0]);
#pragma unroll
      for (int r = 0; r < R; ++r) {
        if (r < n_ch) {
          if (r < P) {
#pragma unroll
            for (int t = 0; t < NT; ++t)
              wr[r][t] = *(const i32x4 *)(smem + lbase + (r * NT + t) * kPkWaves * 1024);
          }
          mac(r);
          if (r + R < n_ch) {
            issue_x(r, r + R);
            issue_w(r, r + R);
          }
        }
        __builtin_amdgcn_sched_barrier(0);
      }
      // steady state: slot r holds chunk c + r and is refilled R chunks ahead
      int c = R;
      for (; c + 2 * R <= n_ch; c += R) {
#pragma unroll
        for (int r = 0; r < R; ++r) {
          mac(r);
          issue_x(r, c + R + r);
          issue_w(r, c + R + r);
          __builtin_amdgcn_sched_barrier(0);
        }
      }
      for (; c < n_ch; c += R) {
#pragma unroll
        for (int r = 0; r < R; ++r) {
          if (c + r < n_ch) {
            mac(r);
            if (c + r + R < n_ch) {
              issue_x(r, c + r + R);
              issue_w(r, c + r + R);
            }
          }
        }
      }

      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
      float *sinv = (float *)(smem + kPkInvOff);  // 1/rms per token
      if (io.scale_rows && gb == t_lo) {
        lds_barrier();
        // 4 threads per token, a quarter of the partial sums each, then the
        // quarters in a fixed order
        const int t = tid() >> 2, qtr = tid() & 3;
        float sum = 0.0f;
        if (t < n_tok) {
          const float *row = (const float *)(smem + kSsOff + t * 1024);
          const int per = (nwg + 3) >> 2;
          const int g0 = qtr * per, g1 = g0 + per < nwg ? g0 + per : nwg;
          for (int g = g0; g < g1; ++g) sum += row[g];
        }
        sum += __shfl_xor(sum, 1, 64);
        sum += __shfl_xor(sum, 2, 64);
        if (t < n_tok && qtr == 0) sinv[t] = 1.0f / sqrtf(sum / (float)a.hidden + a.eps);
      }
      lds_barrier();  // every wave is done with the prefetched chunks; sinv visible
      const float2 *rope = rope_lds ? (const float2 *)stage : a.rope;
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
          const int items = tiles_here * TT * 32;
          for (int it = tid(); it < items; it += kPkThreads) {
            const int tok16 = it & 15, g = (it >> 4) & 1, pr = it >> 5;
            const int tl = pr / TT, tt = pr - tl * TT;
            const int tok = tt * 16 + tok16;
            if (tok < n_tok) {
              const int l1 = tok16 + 16 * g;
              f32x4 v1 = red[0][pr][l1], v2 = red[0][pr][l1 + 32];
#pragma unroll
              for (int ww = 1; ww < kGemmWaves; ++ww) {
                v1 += red[ww][pr][l1];
                v2 += red[ww][pr][l1 + 32];
              }
              if (io.scale_rows) {
                const float rr = sinv[tok];
                v1 *= rr;
                v2 *= rr;
              }
              epilogue(a, io, rope, gb + t0 + tl, 4 * g, tok, v1, v2);
            }
          }
          lds_barrier();
        }
      }
    }
    // a workgroup without tiles still owns its staging loads
    if (t_lo >= t_hi) asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  }

  // Four finished output pairs of tile `tile` (rows p0 + i and p0 + 8 + i,
  // token t), stored with device-scope stores.
  __device__ __forceinline__ void epilogue(const PkArgs &a, const GemmIO &io, const float2 *rope,
                                           int tile, int p0, int t, const f32x4 &v1,
                                           const f32x4 &v2) {
    if constexpr (EPI == EPI_QKV) {
      const int d = a.head_dim, ht = d / 16;
      const int qt = a.n_heads * ht, kt = a.n_kv * ht;
      if (tile < qt + kt) {
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
        const uint2 lo = pack4_bf16(o1[0], o1[1], o1[2], o1[3]);
        const uint2 hi = pack4_bf16(o2[0], o2[1], o2[2], o2[3]);
        if (isq) {
          const __amdgpu_buffer_rsrc_t qrs = rsrc(a.q, (long long)a.n_tok * a.n_heads * d * 2);
          const int off = ((t * a.n_heads + head) * d + j0) * 2;
          __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(__attribute__((ext_vector_type(2))) int, lo), qrs, off, 0, kDev);
          __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(__attribute__((ext_vector_type(2))) int, hi), qrs, off + d, 0, kDev);
        } else {
          const __amdgpu_buffer_rsrc_t krs = rsrc(io.kc, (long long)a.n_kv * a.cap * d * 2);
          const int off = ((head * a.cap + a.kv_len + t) * d + j0) * 2;
          __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(__attribute__((ext_vector_type(2))) int, lo), krs, off, 0, kDev);
          __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(__attribute__((ext_vector_type(2))) int, hi), krs, off + d, 0, kDev);
        }
      } else {
        // V is cached transposed: [head][d][slot]
        const int idx = tile - qt - kt;
        const int head = idx / ht, u = idx % ht;
        const __amdgpu_buffer_rsrc_t vrs = rsrc(io.vc, (long long)a.n_kv * a.cap * d * 2);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int off = ((head * d + 16 * u + p0 + i) * a.cap + a.kv_len + t) * 2;
          __builtin_amdgcn_raw_buffer_store_b16(f2bf(v1[i]), vrs, off, 0, kDev);
          __builtin_amdgcn_raw_buffer_store_b16(f2bf(v2[i]), vrs, off + 8 * a.cap * 2, 0, kDev);
        }
      }
    } else if constexpr (EPI == EPI_RESID || EPI == EPI_LOGITS) {
      // RESID: the K range's slice of the projection, [split][n_tok][hidden];
      // LOGITS: [n_tok][vocab]
      const int n = EPI == EPI_RESID ? a.hidden : a.vocab;
      const int slice = EPI == EPI_RESID ? split : 0;
      const __amdgpu_buffer_rsrc_t ors =
          rsrc(io.out_f, (long long)(EPI == EPI_RESID ? p.split : 1) * a.n_tok * n * 4);
      const int row = (slice * a.n_tok + t) * n;
      const int d1 = tile * 16 + p0, d2 = d1 + 8;
      store4(ors, row, d1, n, v1);
      store4(ors, row, d2, n, v2);
    } else if constexpr (EPI == EPI_SWIGLU) {
      float o[4];
#pragma unroll
      for (int i = 0; i < 4; ++i)
        o[i] = v1[i] * __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(v1[i] * -1.44269504f)) * v2[i];
      const __amdgpu_buffer_rsrc_t ars = rsrc(io.out_b, (long long)((a.n_tok + 15) >> 4) * io.out_ks * 1024);
      const uint2 pk = pack4_bf16(o[0], o[1], o[2], o[3]);
      __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(__attribute__((ext_vector_type(2))) int, pk), ars,
                                            (int)packed_index(t, tile * 8 + p0, io.out_ks) * 2, 0, kDev);
    }
  }

  // Four consecutive floats at columns d .. d + 3 of a row (only those below
  // n), device-scope stores.
  __device__ __forceinline__ void store4(__amdgpu_buffer_rsrc_t rs, int row, int d, int n,
                                         const f32x4 &v) {
    if ((n & 3) == 0 && d + 3 < n) {
      __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(i32x4, v), rs, (row + d) * 4, 0, kDev);
    } else {
#pragma unroll
      for (int i = 0; i < 4; ++i)
        if (d + i < n)
          __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(int, v[i]), rs, (row + d + i) * 4, 0, kDev);
    }
  }
};

// ---------------------------------------------------------------------------
// residual add + RMSNorm partials
// ---------------------------------------------------------------------------

// h += sum of the n_slices delta slices (slice order); xa = bf16(h * g)
// packed (padding columns zero); ss[t][wg] = this workgroup's part of the
// row's sum of squares.  Workgroup wg owns a range of 8-column groups of
// the packed width for every row.
__device__ __forceinline__ void pk_norm(const PkArgs &a, int n_slices, const float *g, char *smem) {
  const int nwg = gridDim.x, wg = bid();
  const int n_tok = a.n_tok, H = a.hidden;
  const int G8 = a.xa_ks * 4;  // 8-column groups of the packed width
  const int g0 = (int)(((long long)G8 * wg) / nwg), g1 = (int)(((long long)G8 * (wg + 1)) / nwg);
  const int ng = g1 - g0;
  float *part = (float *)(smem + kSsOff);  // [64 rows][8] partial sums (ng <= 8)
  const int it = tid();
  const int t = ng > 0 ? it / ng : 0, gi = ng > 0 ? it - t * ng : 0;
  const bool live = ng > 0 && t < n_tok;
  const int k0 = (g0 + gi) * 8;
  float sq = 0.0f;
  if (live) {
    const bool inside = k0 < H;
    const __amdgpu_buffer_rsrc_t hrs = rsrc(a.h, (long long)n_tok * H * 4);
    const __amdgpu_buffer_rsrc_t drs = rsrc(a.delta, (long long)kMaxSplit * n_tok * H * 4);
    const __amdgpu_buffer_rsrc_t grs = rsrc(g, (long long)H * 4);
    const int off = inside ? (t * H + k0) * 4 : n_tok * H * 4;
    f32x4 hv[2], dv[kMaxSplit][2], gv[2];
#pragma unroll
    for (int hh = 0; hh < 2; ++hh) {
      hv[hh] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(hrs, off, hh * 16, kDev));
      gv[hh] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(grs, inside ? k0 * 4 : H * 4, hh * 16, 0));
    }
#pragma unroll
    for (int sl = 0; sl < kMaxSplit; ++sl) {
      const int doff = (inside && sl < n_slices) ? ((sl * n_tok + t) * H + k0) * 4 : kMaxSplit * n_tok * H * 4;
#pragma unroll
      for (int hh = 0; hh < 2; ++hh)
        dv[sl][hh] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(drs, doff, hh * 16, kDev));
    }
    if (n_slices > 0) {
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) {
        f32x4 d = dv[0][hh];
#pragma unroll
        for (int sl = 1; sl < kMaxSplit; ++sl) d += dv[sl][hh];  // missing slices read 0
        hv[hh] += d;
      }
      if (inside) {
        __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(i32x4, hv[0]), hrs, off, 0, kDev);
        __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(i32x4, hv[1]), hrs, off + 16, 0, kDev);
      }
    }
#pragma unroll
    for (int hh = 0; hh < 2; ++hh)
#pragma unroll
      for (int e = 0; e < 4; ++e) sq += hv[hh][e] * hv[hh][e];
    uint16_t v[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = f2bf(hv[e >> 2][e & 3] * gv[e >> 2][e & 3]);
    i32x4 o;
    o[0] = (int)(v[0] | ((uint32_t)v[1] << 16));
    o[1] = (int)(v[2] | ((uint32_t)v[3] << 16));
    o[2] = (int)(v[4] | ((uint32_t)v[5] << 16));
    o[3] = (int)(v[6] | ((uint32_t)v[7] << 16));
    const __amdgpu_buffer_rsrc_t xrs = rsrc(a.xa, (long long)((n_tok + 15) >> 4) * a.xa_ks * 1024);
    __builtin_amdgcn_raw_buffer_store_b128(o, xrs, (int)packed_index(t, k0, a.xa_ks) * 2, 0, kDev);
    part[t * 8 + gi] = sq;
  }
  lds_barrier();
  // the workgroup's groups of each row, in order (0 for a workgroup that
  // owns no columns: the consumers sum every workgroup's entry)
  if (it < n_tok) {
    float s = 0.0f;
    for (int j = 0; j < ng; ++j) s += part[it * 8 + j];
    const __amdgpu_buffer_rsrc_t srs = rsrc(a.ss, (long long)n_tok * kSsGroups * 4);
    __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(int, s), srs, (it * kSsGroups + wg) * 4, 0, kDev);
  }
}

// ---------------------------------------------------------------------------
// attention: one (KV head, key range) item per workgroup
// ---------------------------------------------------------------------------

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
  typedef float f32x2 __attribute__((ext_vector_type(2)));
  const f32x2 v = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));
}
__device__ __forceinline__ float swap_max16(float v) {
  const auto r = __builtin_amdgcn_permlane16_swap(__builtin_bit_cast(uint32_t, v),
                                                  __builtin_bit_cast(uint32_t, v), false, false);
  return fmaxf(__builtin_bit_cast(float, (uint32_t)r[0]), __builtin_bit_cast(float, (uint32_t)r[1]));
}
__device__ __forceinline__ float swap_max32(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__builtin_bit_cast(uint32_t, v),
                                                  __builtin_bit_cast(uint32_t, v), false, false);
  return fmaxf(__builtin_bit_cast(float, (uint32_t)r[0]), __builtin_bit_cast(float, (uint32_t)r[1]));
}
__device__ __forceinline__ float swap_sum16(float v) {
  const auto r = __builtin_amdgcn_permlane16_swap(__builtin_bit_cast(uint32_t, v),
                                                  __builtin_bit_cast(uint32_t, v), false, false);
  return __builtin_bit_cast(float, (uint32_t)r[0]) + __builtin_bit_cast(float, (uint32_t)r[1]);
}
__device__ __forceinline__ float swap_sum32(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__builtin_bit_cast(uint32_t, v),
                                                  __builtin_bit_cast(uint32_t, v), false, false);
  return __builtin_bit_cast(float, (uint32_t)r[0]) + __builtin_bit_cast(float, (uint32_t)r[1]);
}

// Visibility of keys k0 .. k0 + 7 for a row with ancestor mask anc: prefix
// slots visible, tree slot kv_len + j visible when bit j is set, slots >=
// nkeys not.
__device__ __forceinline__ uint32_t vis8(const uint32_t *anc, int k0, int kv_len, int nkeys) {
  uint32_t vis;
  const int jt = k0 - kv_len;
  if (jt + 8 <= 0) {
    vis = 0xffu;
  } else if (jt >= 0) {
    const int wi = jt >> 5, sh = jt & 31;
    const uint64_t win = (uint64_t)anc[wi] | ((uint64_t)(wi < 7 ? anc[wi + 1] : 0u) << 32);
    vis = (uint32_t)(win >> sh) & 0xffu;
  } else {
    const int pre = -jt;
    vis = ((anc[0] << pre) | ((1u << pre) - 1u)) & 0xffu;
  }
  const int valid = nkeys - k0;
  if (valid < 8) vis &= valid > 0 ? (1u << valid) - 1u : 0u;
  return vis;
}

constexpr int kAD = 128;          // head_dim of the persistent kernel
constexpr int kANW = kAD / 16;    // waves: one per 16 output dimensions
constexpr int kASW = 2;           // steps per wave (at most)
constexpr int kAMS = kASW * kANW; // steps of an item (at most)
static_assert(kAMS == kPkAttnMaxSteps, "attention item size");
constexpr int kAKSD = kAD / 32;   // k-steps over head_dim

// The register cache of one item: K of the wave's steps, V^T of all steps.
struct AttnRegs {
  i32x4 kf[kASW][2][kAKSD];
  i32x4 vf[kAMS];
};

// Work item of this workgroup's attention phase: (KV head g, range split).
struct AttnItem {
  int g, split, st0, nst;
  bool live;
};

__device__ __forceinline__ AttnItem attn_item(const PkArgs &a, int item) {
  AttnItem it;
  const int nkeys = a.kv_len + a.n_tok;
  const int n_steps = (nkeys + 31) >> 5;
  it.live = item < a.n_kv * a.n_chunks;
  it.g = item / a.n_chunks;
  it.split = item - it.g * a.n_chunks;
  it.st0 = (n_steps * it.split) / a.n_chunks;
  it.nst = (n_steps * (it.split + 1)) / a.n_chunks - it.st0;
  return it;
}

// K rows of the item into registers (every step, one cache policy: the
// device-scope loads see this layer's tree rows, written in this kernel,
// and cost the prefix rows nothing, which are read once).
__device__ __forceinline__ void attn_load_k(const PkArgs &a, const uint16_t *kc, const AttnItem &it,
                                            AttnRegs &rg) {
  const int w = __builtin_amdgcn_readfirstlane(tid() >> 6);
  const int lane = tid() & 63;
  const int lr = lane & 15, lg = lane >> 4;
  const int nkeys = a.kv_len + a.n_tok;
  const int bytes = a.cap * kAD * 2;
  const __amdgpu_buffer_rsrc_t krs = rsrc(kc + (size_t)it.g * a.cap * kAD, bytes);
#pragma unroll
  for (int u = 0; u < kASW; ++u) {
    const int sl = w + kANW * u;
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int slot = (it.st0 + sl) * 32 + 8 * (lr >> 2) + 4 * i + (lr & 3);
      const int vo = (sl < it.nst && slot < nkeys) ? (slot * kAD + 8 * lg) * 2 : bytes;
#pragma unroll
      for (int ks = 0; ks < kAKSD; ++ks)
        rg.kf[u][i][ks] = __builtin_amdgcn_raw_buffer_load_b128(krs, vo, ks * 64, kDev);
    }
  }
}

// V^T rows of the item (dimensions 16 w + lr, keys 8 lg .. 8 lg + 7 of every
// step), requested once the wave has scored its steps so that they do not
// delay the keys.
__device__ __forceinline__ void attn_load_v(const PkArgs &a, const uint16_t *vc, const AttnItem &it,
                                            AttnRegs &rg) {
  const int w = __builtin_amdgcn_readfirstlane(tid() >> 6);
  const int lane = tid() & 63;
  const int lr = lane & 15, lg = lane >> 4;
  const int nkeys = a.kv_len + a.n_tok;
  const int bytes = a.cap * kAD * 2;
  const __amdgpu_buffer_rsrc_t vrs = rsrc(vc + (size_t)it.g * kAD * a.cap, bytes);
#pragma unroll
  for (int j = 0; j < kAMS; ++j) {
    const int key = (it.st0 + j) * 32 + 8 * lg;
    const int vo = (j < it.nst && key < nkeys) ? ((16 * w + lr) * a.cap + key) * 2 : bytes;
    rg.vf[j] = __builtin_amdgcn_raw_buffer_load_b128(vrs, vo, 0, kDev);
  }
}

// Scores, probabilities (bf16 hi + lo parts) and P.V of one item for every
// block of RT 16-row query tiles; writes the unnormalised partial (row max
// m, row sum l, sum p v) of each query row.  The item's K rows are in
// rg.kf for the first block (later blocks, with grouped queries, read them
// again); V is requested after the first block's scores.
//   1. wave w scores its steps (S^T = K Q^T), masks them, stores the float32
//      scores in LDS and the row max;
//   2. each lane reads back its own scores; after a barrier, p = exp(s - M)
//      against the block max is stored as bf16 hi = bf16(p) and lo =
//      bf16(p - hi) (over the scores' bytes), with the row sums;
//   3. wave w computes dimensions 16 w .. 16 w + 15 of O^T = V^T (P_hi +
//      P_lo)^T over all of the item's keys.
template <int RT>
__device__ __forceinline__ void attn_compute(const PkArgs &a, const uint16_t *kc,
                                             const uint16_t *vc, const AttnItem &it_in,
                                             AttnRegs &rg, char *smem) {
  constexpr int RB = 16 * RT;
  constexpr int KW = 32 * kAMS;
  constexpr int NT = kANW * 64;
  // float32 scores [RB][KW + 4] share their bytes with the two bf16 parts
  // [RB][KW + 8] each of the probabilities
  float(*ssc)[KW + 4] = (float(*)[KW + 4])smem;
  uint16_t(*sp)[KW + 8] = (uint16_t(*)[KW + 8])smem;
  uint16_t(*spl)[KW + 8] = (uint16_t(*)[KW + 8])(smem + RB * (KW + 8) * 2);
  uint16_t(*sq)[kAD + 8] = (uint16_t(*)[kAD + 8])(smem + 2 * RB * (KW + 8) * 2);
  uint32_t(*sanc)[8] = (uint32_t(*)[8])(smem + 2 * RB * (KW + 8) * 2 + RB * (kAD + 8) * 2);
  float(*smax)[RB] = (float(*)[RB])((char *)sanc + RB * 8 * 4);
  float(*ssum)[RB] = (float(*)[RB])((char *)smax + kANW * RB * 4);
  static_assert(RB * (KW + 4) * 4 <= 2 * RB * (KW + 8) * 2, "scores fit the probability buffers");

  const int G = a.n_heads / a.n_kv;
  const float inv_g = 1.0f / (float)G;
  const int R = a.n_tok * G;
  const int nkeys = a.kv_len + a.n_tok;
  const int qbytes = a.n_tok * a.n_heads * kAD * 2;
  const __amdgpu_buffer_rsrc_t qrs = rsrc(a.q, qbytes);
  const int abytes = a.n_tok * 8 * 4;
  const __amdgpu_buffer_rsrc_t ars = rsrc(a.meta->anc, abytes);
  const float c = a.scale * 1.44269504088896340736f;
  const int pbytes = a.n_kv * a.n_chunks * R * kAD * 4;
  const __amdgpu_buffer_rsrc_t pors = rsrc(a.part_o, pbytes);
  const __amdgpu_buffer_rsrc_t pmrs = rsrc(a.part_ml, a.n_kv * a.n_chunks * R * 8);

  for (int rb0 = 0; rb0 < R; rb0 += RB) {
    // the item and block values are re-read each block (opaque), so that
    // nothing derived from them is hoisted out of this loop and held
    // across it
    const int rb = sopaque(rb0);
    AttnItem it;
    it.g = sopaque(it_in.g);
    it.split = sopaque(it_in.split);
    it.st0 = sopaque(it_in.st0);
    it.nst = sopaque(it_in.nst);
    it.live = true;
    const int w = __builtin_amdgcn_readfirstlane(tid() >> 6);
    const int lane = tid() & 63;
    const int lr = lane & 15, lg = lane >> 4;
    if (rb > 0) attn_load_k(a, kc, it, rg);  // K again for a later block of grouped queries
    // ---- stage the block's query rows and ancestor masks
    constexpr int QPT = (RB * (kAD / 8) + NT - 1) / NT;
#pragma unroll
    for (int j = 0; j < QPT; ++j) {
      const int idx = tid() + j * NT;
      const int rr = idx / (kAD / 8), d0 = (idx % (kAD / 8)) * 8;
      const int r = rb + rr;
      const int t = (int)(((float)r + 0.5f) * inv_g), hl = r - t * G;
      const int vo = (rr < RB && r < R) ? ((t * a.n_heads + it.g * G + hl) * kAD + d0) * 2 : qbytes;
      const i32x4 v = __builtin_amdgcn_raw_buffer_load_b128(qrs, vo, 0, kDev);
      if (rr < RB) *(i32x4 *)&sq[rr][d0] = v;
    }
    for (int idx = tid(); idx < RB * 8; idx += NT) {
      const int rr = idx >> 3, wd = idx & 7;
      const int r = rb + rr;
      const int t = (int)(((float)r + 0.5f) * inv_g);
      const int vo = r < R ? (t * 8 + wd) * 4 : abytes;
      sanc[rr][wd] = (uint32_t)__builtin_amdgcn_raw_buffer_load_b32(ars, vo, 0, 0);
    }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");  // the staging loads (and the K rows)
    lds_barrier();

    // ---- 1. scores of the wave's steps into LDS, row max
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
      float mx = -INFINITY;
#pragma unroll
      for (int u = 0; u < kASW; ++u) {
        __builtin_amdgcn_sched_barrier(0);
        const int sl = w + kANW * u;
        const int k0 = (it.st0 + sl) * 32 + 8 * lg;  // this lane's 8 keys of the step
        f32x4 sacc[2] = {f32x4{0.f, 0.f, 0.f, 0.f}, f32x4{0.f, 0.f, 0.f, 0.f}};
#pragma unroll
        for (int ks = 0; ks < kAKSD; ++ks) {
          const uint4 qv = *(const uint4 *)&sq[rt * 16 + lr][32 * ks + 8 * lg];
#pragma unroll
          for (int i = 0; i < 2; ++i)
            sacc[i] = mfma16(__builtin_bit_cast(bf16x8, rg.kf[u][i][ks]), as_bf16x8(qv), sacc[i]);
        }
        // element e of sacc[i]: key k0 + 4 i + e, row rb + 16 rt + lr
        float sv[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) sv[j] = sacc[j >> 2][j & 3];
        if (sl >= it.nst) {
#pragma unroll
          for (int j = 0; j < 8; ++j) sv[j] = -INFINITY;
        } else if ((it.st0 + sl + 1) * 32 > a.kv_len) {
          const uint32_t vis = vis8(sanc[rt * 16 + lr], k0, a.kv_len, nkeys);
#pragma unroll
          for (int j = 0; j < 8; ++j) sv[j] = (vis >> j) & 1u ? sv[j] : -INFINITY;
        }
        f32x4 *dst = (f32x4 *)&ssc[rt * 16 + lr][32 * sl + 8 * lg];
        dst[0] = f32x4{sv[0], sv[1], sv[2], sv[3]};
        dst[1] = f32x4{sv[4], sv[5], sv[6], sv[7]};
        mx = fmaxf(mx, fmaxf(fmaxf(fmaxf(sv[0], sv[1]), fmaxf(sv[2], sv[3])),
                             fmaxf(fmaxf(sv[4], sv[5]), fmaxf(sv[6], sv[7]))));
      }
      mx = swap_max32(swap_max16(mx));
      if (lg == 0) smax[w][rt * 16 + lr] = mx;
    }
    if (rb == 0) {
      __builtin_amdgcn_sched_barrier(0);
      attn_load_v(a, vc, it, rg);
      __builtin_amdgcn_sched_barrier(0);
    }
    lds_barrier();

    // ---- 2. probabilities against the block max (hi + lo bf16 parts), row sums
    {
      f32x4 sv[RT][kASW][2];
#pragma unroll
      for (int rt = 0; rt < RT; ++rt)
#pragma unroll
        for (int u = 0; u < kASW; ++u) {
          const f32x4 *src = (const f32x4 *)&ssc[rt * 16 + lr][32 * (w + kANW * u) + 8 * lg];
          sv[rt][u][0] = src[0];
          sv[rt][u][1] = src[1];
        }
      float Mc[RT];
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) {
        const int rr = rt * 16 + lr;
        float M = smax[0][rr];
#pragma unroll
        for (int ww = 1; ww < kANW; ++ww) M = fmaxf(M, smax[ww][rr]);
        Mc[rt] = (M == -INFINITY ? 0.0f : M) * c;
      }
      lds_barrier();  // every lane holds its scores: their bytes are free
#pragma unroll
      for (int rt = 0; rt < RT; ++rt) {
        const int rr = rt * 16 + lr;
        float ps = 0.0f;
#pragma unroll
        for (int u = 0; u < kASW; ++u) {
          const int sl = w + kANW * u;
          float pv[8];
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            pv[j] = __builtin_amdgcn_exp2f(fmaf(sv[rt][u][j >> 2][j & 3], c, -Mc[rt]));
            ps += pv[j];
          }
          uint32_t hi[4], lo[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            hi[e] = pack_bf16x2(pv[2 * e], pv[2 * e + 1]);
            lo[e] = pack_bf16x2(pv[2 * e] - __uint_as_float(hi[e] << 16),
                                pv[2 * e + 1] - __uint_as_float(hi[e] & 0xffff0000u));
          }
          *(uint4 *)&sp[rr][32 * sl + 8 * lg] = make_uint4(hi[0], hi[1], hi[2], hi[3]);
          *(uint4 *)&spl[rr][32 * sl + 8 * lg] = make_uint4(lo[0], lo[1], lo[2], lo[3]);
        }
        ps = swap_sum32(swap_sum16(ps));
        if (lg == 0) ssum[w][rr] = ps;
      }
    }
    lds_barrier();

    // ---- 3. O^T for dimensions 16 w .. 16 w + 15 over all of the keys.
    // The lane's byte offset in the probability arrays is taken here (an
    // opaque value) so that every read below is that base plus a constant,
    // instead of one address register per (step, tile) hoisted out of the
    // row-block loop.
    f32x4 oacc[RT];
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) oacc[rt] = f32x4{0.f, 0.f, 0.f, 0.f};
    {
      constexpr int ROW = (KW + 8) * 2;  // bytes per row of sp / spl
      const int pb = vopaque((tid() & 15) * ROW + ((tid() & 63) >> 4) * 16);
      const char *php = smem + pb;
      const char *plp = smem + RB * ROW + pb;
#pragma unroll
      for (int j = 0; j < kAMS; ++j) {
        if (j < it.nst) {
          i32x4 vv = rg.vf[j];
          if ((it.st0 + j + 1) * 32 > nkeys) {  // the step passes the last key (wave-uniform)
            // slots never written for this step: zero (their probabilities
            // are zero, but the bits there need not be a finite number)
            const int valid = vopaque(nkeys - (it.st0 + j) * 32 - 8 * lg);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              const uint32_t lo = 2 * e < valid ? 0x0000ffffu : 0u;
              const uint32_t hi = 2 * e + 1 < valid ? 0xffff0000u : 0u;
              vv[e] &= (int)(lo | hi);
            }
          }
#pragma unroll
          for (int rt = 0; rt < RT; ++rt) {
            const uint4 pf = *(const uint4 *)(php + rt * 16 * ROW + 64 * j);
            const uint4 pl = *(const uint4 *)(plp + rt * 16 * ROW + 64 * j);
            oacc[rt] = mfma16(__builtin_bit_cast(bf16x8, vv), as_bf16x8(pf), oacc[rt]);
            oacc[rt] = mfma16(__builtin_bit_cast(bf16x8, vv), as_bf16x8(pl), oacc[rt]);
          }
        }
        __builtin_amdgcn_sched_barrier(0);
      }
    }
    const int base = (it.g * a.n_chunks + it.split) * R;
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
      const int r = rb + rt * 16 + lr;
      if (r < R)
        __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(i32x4, oacc[rt]), pors,
                                               ((base + r) * kAD + 16 * w + 4 * lg) * 4, 0, kDev);
    }
    if (tid() < RB) {
      const int rr = tid();
      const int r = rb + rr;
      if (r < R) {
        float M = smax[0][rr], L = ssum[0][rr];
#pragma unroll
        for (int ww = 1; ww < kANW; ++ww) {
          M = fmaxf(M, smax[ww][rr]);
          L += ssum[ww][rr];
        }
        typedef int i32x2 __attribute__((ext_vector_type(2)));
        const i32x2 ml = {__builtin_bit_cast(int, M == -INFINITY ? M : M * a.scale),
                          __builtin_bit_cast(int, L)};
        __builtin_amdgcn_raw_buffer_store_b64(ml, pmrs, (base + r) * 8, 0, kDev);
      }
    }
    lds_barrier();  // LDS free for the next row block
  }
}

// ---------------------------------------------------------------------------
// merge of the key ranges: one thread per (row t, query head, 8 dimensions)
// ---------------------------------------------------------------------------

constexpr int kMergeGroup = 8;  // key ranges loaded per round trip

// Every load of a group of 8 ranges (statistics and the thread's 8
// dimensions) is issued before any use; groups after the first rescale the
// running sums to the new maximum (one group when n_chunks <= 8).
__device__ __forceinline__ void pk_merge(const PkArgs &a) {
  constexpr int TPP = kAD / 8;
  const int nc = a.n_chunks;
  const int G = a.n_heads / a.n_kv;
  const int R = a.n_tok * G;
  const int mbytes = a.n_kv * nc * R * 8;
  const int obytes = a.n_kv * nc * R * kAD * 4;
  const __amdgpu_buffer_rsrc_t mrs = rsrc(a.part_ml, mbytes);
  const __amdgpu_buffer_rsrc_t ors = rsrc(a.part_o, obytes);
  const int xbytes = ((a.n_tok + 15) >> 4) * a.xo_ks * 1024;
  const __amdgpu_buffer_rsrc_t xrs = rsrc(a.xo, xbytes);
  const int total = a.n_tok * a.n_heads * TPP;
  for (int base = bid() * kPkThreads; base < total; base += gridDim.x * kPkThreads) {
    const int gid = base + (int)tid();
    const bool live = gid < total;
    const int pair = gid / TPP, part = gid - pair * TPP;
    const int t = pair / a.n_heads, head = pair - t * a.n_heads;
    const int g = head / G;
    const int r = t * G + (head - g * G);
    float M = -INFINITY, L = 0.0f;
    f32x4 o0 = {0.f, 0.f, 0.f, 0.f}, o1 = {0.f, 0.f, 0.f, 0.f};
    for (int c0 = 0; c0 < nc; c0 += kMergeGroup) {
      float2 st[kMergeGroup];
      f32x4 lo[kMergeGroup], hi[kMergeGroup];
#pragma unroll
      for (int k = 0; k < kMergeGroup; ++k) {
        const int cc = c0 + k;
        const int row = (g * nc + cc) * R + r;
        const bool in = live && cc < nc;
        const int mo = in ? row * 8 : mbytes;
        const int oo = in ? (row * kAD + part * 8) * 4 : obytes;
        st[k].x = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(mrs, mo, 0, kDev));
        st[k].y = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(mrs, mo + 4, 0, kDev));
        lo[k] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(ors, oo, 0, kDev));
        hi[k] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(ors, oo + 16, 0, kDev));
      }
#pragma unroll
      for (int k = 0; k < kMergeGroup; ++k)
        if (c0 + k >= nc) st[k].x = -INFINITY;
      float Mn = M;
#pragma unroll
      for (int k = 0; k < kMergeGroup; ++k) Mn = fmaxf(Mn, st[k].x);
      const float sc = M == -INFINITY ? 0.0f : expf(M - Mn);
      L *= sc;
      o0 *= sc;
      o1 *= sc;
#pragma unroll
      for (int k = 0; k < kMergeGroup; ++k) {
        const float wgt = st[k].x == -INFINITY ? 0.0f : expf(st[k].x - Mn);
        L += wgt * st[k].y;
        o0 += wgt * lo[k];
        o1 += wgt * hi[k];
      }
      M = Mn;
    }
    const float inv = 1.0f / L;
    i32x4 pk;
    pk[0] = (int)(f2bf(o0[0] * inv) | ((uint32_t)f2bf(o0[1] * inv) << 16));
    pk[1] = (int)(f2bf(o0[2] * inv) | ((uint32_t)f2bf(o0[3] * inv) << 16));
    pk[2] = (int)(f2bf(o1[0] * inv) | ((uint32_t)f2bf(o1[1] * inv) << 16));
    pk[3] = (int)(f2bf(o1[2] * inv) | ((uint32_t)f2bf(o1[3] * inv) << 16));
    if (live) {
      __builtin_amdgcn_raw_buffer_store_b128(pk, xrs, (int)packed_index(t, head * kAD + part * 8, a.xo_ks) * 2,
                                             0, kDev);
      // the last head's threads clear the row's padding columns
      if (head == a.n_heads - 1) {
        for (int k0 = a.n_heads * kAD + part * 8; k0 < a.xo_ks * 32; k0 += TPP * 8)
          __builtin_amdgcn_raw_buffer_store_b128(i32x4{0, 0, 0, 0}, xrs,
                                                 (int)packed_index(t, k0, a.xo_ks) * 2, 0, kDev);
      }
    }
  }
}

// ---------------------------------------------------------------------------
// the kernel
// ---------------------------------------------------------------------------

// A GEMM stage: the first pass's prefetch (waves 1..7), barrier, the
// optional light phase `mid` (every wave, then a second barrier), the GEMM.
// Returns false if a barrier failed.
template <int EPI, int TT, int NT, typename Mid>
__device__ __forceinline__ bool gemm_stage(const PkArgs &a, const PkGemmPlan &pl, const GemmIO &io, char *smem,
                           unsigned &bi, int *s_ok, bool has_mid, Mid &&mid) {
  PkGemm<EPI, TT, NT> G;
  G.plan(pl);
  const int w = __builtin_amdgcn_readfirstlane(tid() >> 6);
  pk_drain();
  if (w != 0) G.prefetch(io.W, G.t_lo, smem);
  if (!pk_wait(a.sync, bi, s_ok)) return false;
  if (has_mid) {
    mid();
    pk_drain();
    if (!pk_wait(a.sync, bi, s_ok)) return false;
  }
  G.run(a, io, smem, true);
  return true;
}

// Tiles per pass of each GEMM of a layer and of the LM head.
template <int TT_, int RT_, int NQ, int NO, int NG, int ND, int NL>
struct PkSig {
  static constexpr int TT = TT_, RT = RT_, NT_QKV = NQ, NT_O = NO, NT_GU = NG, NT_DN = ND,
                       NT_LM = NL;
};

// The attention of one layer: the first item's prefix K/V requested before
// the barrier (waves 1..7), then every item of this workgroup.
template <int RT>
__device__ __forceinline__ bool attn_stage(const PkArgs &a, const uint16_t *kc, const uint16_t *vc,
                                           char *smem, unsigned &bi, int *s_ok) {
  const int w = __builtin_amdgcn_readfirstlane(tid() >> 6);
  const int n_items = a.n_kv * a.n_chunks;
  {
    AttnRegs rg;
    const AttnItem it = attn_item(a, bid());
    // an item whose keys all lie in the committed prefix (not written in
    // this kernel) requests them before the barrier, in waves 1..7
    const bool early = it.live && w != 0 && (it.st0 + it.nst) * 32 <= a.kv_len;
    pk_drain();
    if (early) attn_load_k(a, kc, it, rg);
    if (!pk_wait(a.sync, bi, s_ok)) return false;
    if (it.live) {
      if (!early) attn_load_k(a, kc, it, rg);
      attn_compute<RT>(a, kc, vc, it, rg, smem);
    }
  }
  for (int item = bid() + gridDim.x; item < n_items; item += gridDim.x) {
    AttnRegs rg;
    const AttnItem it = attn_item(a, item);
    attn_load_k(a, kc, it, rg);
    attn_compute<RT>(a, kc, vc, it, rg, smem);
  }
  return true;
}

// The kernel's arguments through a pointer the compiler cannot see through:
// every stage re-reads the fields it uses from the argument segment instead
// of keeping all of them in scalar registers across the whole forward.
typedef const __attribute__((address_space(4))) PkArgs *PkArgsPtr;
__device__ __forceinline__ const PkArgs &fresh(PkArgsPtr p) {
  asm volatile("" : "+s"(p));
  return *(const PkArgs *)p;
}

template <typename S>
__global__ __launch_bounds__(kPkThreads, 1) void k_persist(PkArgs args) {
  constexpr int TT = S::TT;
  // the arguments in the kernel-argument segment (the only argument, at
  // offset 0); read through this pointer, never copied
  const PkArgsPtr ap = (PkArgsPtr)__builtin_amdgcn_kernarg_segment_ptr();
  __shared__ __attribute__((aligned(16))) char smem[kPkLds];
  int *s_ok = (int *)(smem + kPkOkOff);
  unsigned bi = 0;
  auto nothing = [] {};

  // layer 0's input norm: h is the embedding (no slices)
  {
    const PkArgs &a = fresh(ap);
    pk_norm(a, 0, a.layers[0].g_attn, smem);
  }
  const int n_layers = fresh(ap).n_layers;
  for (int l = 0; l < n_layers; ++l) {
    // ---- [residual + this layer's input norm,] QKV; the first weights are
    // prefetched before the barrier that precedes the norm
    {
      const PkArgs &a = fresh(ap);
      const PkLayer lw = a.layers[l];
      GemmIO io{};
      io.W = lw.qkv;
      io.X = a.xa;
      io.scale_rows = 1;
      io.kc = a.kc + (size_t)l * a.layer_kv;
      io.vc = a.vc + (size_t)l * a.layer_kv;
      if (!gemm_stage<EPI_QKV, TT, S::NT_QKV>(a, a.qkv, io, smem, bi, s_ok, l > 0, [&] {
            const PkArgs &b = fresh(ap);
            pk_norm(b, b.dn.split, b.layers[l].g_attn, smem);
          }))
        return;
    }
    // ---- attention
    {
      const PkArgs &a = fresh(ap);
      if (!attn_stage<S::RT>(a, a.kc + (size_t)l * a.layer_kv, a.vc + (size_t)l * a.layer_kv, smem,
                             bi, s_ok))
        return;
    }
    // ---- range merge, then O
    {
      const PkArgs &a = fresh(ap);
      GemmIO io{};
      io.W = a.layers[l].o;
      io.X = a.xo;
      io.out_f = a.delta;
      if (!gemm_stage<EPI_RESID, TT, S::NT_O>(a, a.o, io, smem, bi, s_ok, true,
                                               [&] { pk_merge(fresh(ap)); }))
        return;
    }
    // ---- residual + post-attention norm, then gate/up
    {
      const PkArgs &a = fresh(ap);
      GemmIO io{};
      io.W = a.layers[l].gu;
      io.X = a.xa;
      io.scale_rows = 1;
      io.out_b = a.act;
      io.out_ks = a.act_ks;
      if (!gemm_stage<EPI_SWIGLU, TT, S::NT_GU>(a, a.gu, io, smem, bi, s_ok, true, [&] {
            const PkArgs &b = fresh(ap);
            pk_norm(b, b.o.split, b.layers[l].g_mlp, smem);
          }))
        return;
    }
    // ---- down
    {
      const PkArgs &a = fresh(ap);
      GemmIO io{};
      io.W = a.layers[l].dn;
      io.X = a.act;
      io.out_f = a.delta;
      if (!gemm_stage<EPI_RESID, TT, S::NT_DN>(a, a.dn, io, smem, bi, s_ok, false, nothing))
        return;
    }
  }
  // ---- residual + final norm, then the LM head
  {
    const PkArgs &a = fresh(ap);
    GemmIO io{};
    io.W = a.lm_head;
    io.X = a.xa;
    io.scale_rows = 1;
    io.out_f = a.logits;
    gemm_stage<EPI_LOGITS, TT, S::NT_LM>(a, a.lm, io, smem, bi, s_ok, true, [&] {
      const PkArgs &b = fresh(ap);
      pk_norm(b, b.dn.split, b.g_final, smem);
    });
  }
}

}  // namespace
}  // namespace sb
