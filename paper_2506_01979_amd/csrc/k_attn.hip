// Branch-masked attention over a shared prefix KV cache (bf16, matrix cores).
//
// Every tree row attends to the committed prefix (cache slots [0, kv_len))
// and to the tree rows on its own path root..i (slots kv_len + j with bit j
// of its ancestor mask) -- the branch-causal mask under which one forward
// scores all branches at once while each branch sees exactly what a separate
// causal forward of that branch would see (Section "Branch Resampling").
//
// Flash-decoding split: the key range [0, kv_len + n_tok) of each KV head is
// cut into n_chunks ranges of at most 2 NW 32-key steps (NW = head_dim / 16
// waves per workgroup); a workgroup takes one range and one block of at
// most 48 query rows of the KV head's group (with grouped queries a head's
// group has n_tok G rows; the workgroups of one range sit on one XCD, so
// its K and V come from HBM once and from that XCD's L2 after).  About one
// workgroup per compute unit.  The workgroup reads its K rows and rows of
// the transposed V cache straight into registers and scores its row block:
//   1. wave w scores steps w and w + NW: S^T = K Q^T, masked, row max into
//      LDS;
//   2. after a barrier, the block max M of each row gives p = exp(s - M);
//      the wave writes its probabilities and their row sums to LDS, each
//      probability as two bf16 parts, hi = bf16(p) and lo = bf16(p - hi),
//      so the matrix-core product below sees p to about 16 bits (the
//      probabilities are not a bf16 rounding point of the forward);
//   3. after a barrier, wave w computes the 16 dimensions 16 w .. 16 w + 15
//      of O^T = V^T P^T = V^T P_hi^T + V^T P_lo^T over all of the
//      workgroup's keys, reading P from LDS, and writes them: every output
//      element is finished by one wave, so the waves never merge
//      accumulators.
// K rows are fetched in a permuted order so that lane group lg of S^T holds
// keys 8 lg .. 8 lg + 7, the layout P is stored and read back in.  The
// workgroup writes an unnormalised partial (row max m, row sum l, sum p v)
// per query row; the merge kernel combines the ranges with the log-sum-exp
// rule.
#include <math.h>

#include "sb_device.h"
#include "sb_internal_fwd.h"

namespace sb {
namespace {

// Workgroup barrier for LDS traffic only (does not wait for global loads).
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// Two floats to packed bf16 (round to nearest even), one instruction.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
  typedef float f32x2 __attribute__((ext_vector_type(2)));
  const f32x2 v = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));
}

// Max / sum over the lane pairs (l, l ^ 16) and (l, l ^ 32) with the gfx950
// lane-swap instructions: swapping a value with itself yields, in every lane,
// the pair's even-row and odd-row values.
__device__ __forceinline__ float max_x16(float v) {
  const auto r = __builtin_amdgcn_permlane16_swap(__builtin_bit_cast(uint32_t, v),
                                                  __builtin_bit_cast(uint32_t, v), false, false);
  return fmaxf(__builtin_bit_cast(float, (uint32_t)r[0]), __builtin_bit_cast(float, (uint32_t)r[1]));
}
__device__ __forceinline__ float max_x32(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__builtin_bit_cast(uint32_t, v),
                                                  __builtin_bit_cast(uint32_t, v), false, false);
  return fmaxf(__builtin_bit_cast(float, (uint32_t)r[0]), __builtin_bit_cast(float, (uint32_t)r[1]));
}
__device__ __forceinline__ float sum_x16(float v) {
  const auto r = __builtin_amdgcn_permlane16_swap(__builtin_bit_cast(uint32_t, v),
                                                  __builtin_bit_cast(uint32_t, v), false, false);
  return __builtin_bit_cast(float, (uint32_t)r[0]) + __builtin_bit_cast(float, (uint32_t)r[1]);
}
__device__ __forceinline__ float sum_x32(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__builtin_bit_cast(uint32_t, v),
                                                  __builtin_bit_cast(uint32_t, v), false, false);
  return __builtin_bit_cast(float, (uint32_t)r[0]) + __builtin_bit_cast(float, (uint32_t)r[1]);
}

// Visibility of the 8 keys k0 .. k0 + 7 (k0 a multiple of 8) for a row with
// ancestor mask anc (LDS): prefix slots are visible, tree slot kv_len + j is
// visible when bit j is set, slots >= nkeys are not.
__device__ __forceinline__ uint32_t visible8(const uint32_t *anc, int k0, int kv_len, int nkeys) {
  uint32_t vis;
  const int jt = k0 - kv_len;
  if (jt + 8 <= 0) {
    vis = 0xffu;
  } else if (jt >= 0) {
    const int wi = jt >> 5, sh = jt & 31;  // bits jt .. jt + 7 of the 256-bit mask
    const uint64_t win = (uint64_t)anc[wi] | ((uint64_t)(wi < 7 ? anc[wi + 1] : 0u) << 32);
    vis = (uint32_t)(win >> sh) & 0xffu;
  } else {
    const int pre = -jt;  // 1..7 prefix keys, then tree bits 0 ..
    vis = ((anc[0] << pre) | ((1u << pre) - 1u)) & 0xffu;
  }
  const int valid = nkeys - k0;
  if (valid < 8) vis &= valid > 0 ? (1u << valid) - 1u : 0u;
  return vis;
}

// D: head_dim; RT: 16-row query tiles per row block; SW: 32-key steps per
// wave (at most).  SW = 1 halves the keys, registers and LDS of a workgroup
// so that two fit on a compute unit (launches of more workgroups than
// compute units: one workgroup's scoring overlaps another's loads).
// LOOP: the workgroup walks every row block of its key range (the launch
// does not split the row blocks); otherwise it scores one.
template <int D, int RT, int SW, bool LOOP>
__global__ __launch_bounds__(D * 4, SW == 1 ? 4 : 2) void k_attn(AttnArgs a) {
  constexpr int NW = D / 16;   // waves: one per 16 output dimensions
  constexpr int NT = NW * 64;
  constexpr int KSD = D / 32;  // k-steps over head_dim (S)
  constexpr int RB = 16 * RT;  // rows per block
  constexpr int MS = SW * NW;  // steps of a workgroup (at most)
  constexpr int KW = 32 * MS;  // keys of a workgroup (at most)
  __shared__ uint16_t sp[RB][KW + 8];  // probabilities, bf16 high part, row-major
  __shared__ uint16_t spl[RB][KW + 8]; // probabilities, bf16 low part
  __shared__ uint16_t sq[RB][D + 8];   // query rows of the block (bf16)
  __shared__ uint32_t sanc[RB][8];
  __shared__ float smax[NW][RB];
  __shared__ float ssum[NW][RB];

  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  const int lr = lane & 15, lg = lane >> 4;
  const int G = a.n_heads / a.n_kv;
  const float inv_g = 1.0f / (float)G;  // r / G = floor((r + 0.5) / G) for r < 2^20
  const int R = a.n_tok * G;
  // Work unit (KV head g, key range split, row block), or (g, split) with
  // every row block in turn when the launch does not split the row blocks
  // (a.rb_split = 0).  Units are numbered XCD-major (workgroup b runs on
  // XCD b % 8) with the row block fastest, so the workgroups that read the
  // same key range sit on one XCD and share its L2.
  const int n_rb = LOOP ? 1 : (R + RB - 1) / RB;
  const int nb = gridDim.x;
  const int unit = (nb & 7) == 0 ? (blockIdx.x & 7) * (nb >> 3) + (blockIdx.x >> 3) : blockIdx.x;
  const int rb0 = (unit % n_rb) * RB;
  const int g = unit / n_rb / a.n_chunks, split = unit / n_rb % a.n_chunks;
  const int nkeys = a.kv_len + a.n_tok;
  const int n_steps = (nkeys + 31) >> 5;
  const int st0 = (n_steps * split) / a.n_chunks, st1 = (n_steps * (split + 1)) / a.n_chunks;
  const int nst = st1 - st0;  // 1 .. MS
  const int kbytes = a.cap * D * 2, vbytes = kbytes;  // one head's K (or V^T) block
  const __amdgpu_buffer_rsrc_t krs = __builtin_amdgcn_make_buffer_rsrc(
      (void *)((const uint16_t *)a.kc + (size_t)g * a.cap * D), 0, kbytes, kBufferDword3);
  const __amdgpu_buffer_rsrc_t vrs = __builtin_amdgcn_make_buffer_rsrc(
      (void *)((const uint16_t *)a.vc + (size_t)g * D * a.cap), 0, vbytes, kBufferDword3);
  const int qbytes = a.n_tok * a.n_heads * D * 2;
  const __amdgpu_buffer_rsrc_t qrs =
      __builtin_amdgcn_make_buffer_rsrc((void *)a.q, 0, qbytes, kBufferDword3);
  const int abytes = a.n_tok * 8 * 4;  // ancestor words of the step's rows
  const __amdgpu_buffer_rsrc_t ars =
      __builtin_amdgcn_make_buffer_rsrc((void *)a.meta->anc, 0, abytes, kBufferDword3);
  // exp(x * scale) = exp2(x * c): one FMA per score before the exp2
  const float c = a.scale * 1.44269504088896340736f;

  // The staging loads of a row block (query rows, ancestor masks) go out
  // before the cache reads: in-order completion lets the staging wait cover
  // only them.
  constexpr int QPT = (RB * (D / 8) + NT - 1) / NT;
  constexpr int APT = (RB * 8 + NT - 1) / NT;
  i32x4 qst[QPT];
  int ast[APT];
  auto stage_loads = [&](int rb) {
#pragma unroll
    for (int j = 0; j < QPT; ++j) {
      const int idx = threadIdx.x + j * NT;
      const int rr = idx / (D / 8), d0 = (idx % (D / 8)) * 8;
      const int r = rb + rr;
      const int t = (int)(((float)r + 0.5f) * inv_g), hl = r - t * G;
      const int vo = (rr < RB && r < R) ? ((t * a.n_heads + g * G + hl) * D + d0) * 2 : qbytes;
      qst[j] = __builtin_amdgcn_raw_buffer_load_b128(qrs, vo, 0, 0);
    }
#pragma unroll
    for (int j = 0; j < APT; ++j) {
      const int idx = threadIdx.x + j * NT;
      const int rr = idx >> 3, wd = idx & 7;
      const int r = rb + rr;
      const int t = (int)(((float)r + 0.5f) * inv_g);
      const int vo = (rr < RB && r < R) ? (t * 8 + wd) * 4 : abytes;
      ast[j] = __builtin_amdgcn_raw_buffer_load_b32(ars, vo, 0, 0);
    }
  };
  stage_loads(rb0);
  __builtin_amdgcn_sched_barrier(0);  // issue order: staging, K (V after scoring)

  // ---- the workgroup's cache reads, once, into registers.  Lanes whose
  // slot is >= nkeys (or past the workgroup's steps) get an offset past the
  // end of the head's buffer and read zero.
  // K: the wave's steps w + NW u; row rho of key tile i is key
  // 8 (rho / 4) + 4 i + rho % 4
  i32x4 kf[SW][2][KSD];
#pragma unroll
  for (int u = 0; u < SW; ++u) {
    const int sl = w + NW * u;
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int slot = (st0 + sl) * 32 + 8 * (lr >> 2) + 4 * i + (lr & 3);
      const int vo = (sl < nst && slot < nkeys) ? (slot * D + 8 * lg) * 2 : kbytes;
#pragma unroll
      for (int ks = 0; ks < KSD; ++ks)
        kf[u][i][ks] = __builtin_amdgcn_raw_buffer_load_b128(krs, vo, ks * 64, 0);
    }
  }
  __builtin_amdgcn_sched_barrier(0);
  // V^T (dimensions 16 w + lr, keys 8 lg .. 8 lg + 7 of every step j) is
  // requested once the wave has scored its steps: issued with K, its
  // requests delayed the keys the scoring waits for
  i32x4 vf[MS];

  // one block of query rows (its staging loads already issued)
  auto row_block = [&](int rb, bool first) {
    // ---- stage the block's query rows and ancestor masks
#pragma unroll
    for (int j = 0; j < QPT; ++j) {
      const int idx = threadIdx.x + j * NT;
      const int rr = idx / (D / 8), d0 = (idx % (D / 8)) * 8;
      if (rr < RB) *(i32x4 *)&sq[rr][d0] = qst[j];
    }
#pragma unroll
    for (int j = 0; j < APT; ++j) {
      const int idx = threadIdx.x + j * NT;
      if ((idx >> 3) < RB) sanc[idx >> 3][idx & 7] = (uint32_t)ast[j];
    }
    lds_barrier();

    // ---- 1. scores of the wave's steps, row max
    float sv[SW][RT][8];
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
      float mx = -INFINITY;
#pragma unroll
      for (int u = 0; u < SW; ++u) {
        const int sl = w + NW * u;
        const int k0 = (st0 + sl) * 32 + 8 * lg;  // this lane's 8 keys of the step
        f32x4 sacc[2] = {f32x4{0.f, 0.f, 0.f, 0.f}, f32x4{0.f, 0.f, 0.f, 0.f}};
#pragma unroll
        for (int ks = 0; ks < KSD; ++ks) {
          const uint4 qv = *(const uint4 *)&sq[rt * 16 + lr][32 * ks + 8 * lg];
#pragma unroll
          for (int i = 0; i < 2; ++i)
            sacc[i] = mfma16(__builtin_bit_cast(bf16x8, kf[u][i][ks]), as_bf16x8(qv), sacc[i]);
        }
        // element e of sacc[i]: key k0 + 4 i + e, row rb + 16 rt + lr
#pragma unroll
        for (int j = 0; j < 8; ++j) sv[u][rt][j] = sacc[j >> 2][j & 3];
        if (sl >= nst) {
#pragma unroll
          for (int j = 0; j < 8; ++j) sv[u][rt][j] = -INFINITY;
        } else if ((st0 + sl + 1) * 32 > a.kv_len) {  // the step reaches past the prefix
          const uint32_t vis = visible8(sanc[rt * 16 + lr], k0, a.kv_len, nkeys);
#pragma unroll
          for (int j = 0; j < 8; ++j) sv[u][rt][j] = (vis >> j) & 1u ? sv[u][rt][j] : -INFINITY;
        }
        mx = fmaxf(mx, fmaxf(fmaxf(fmaxf(sv[u][rt][0], sv[u][rt][1]), fmaxf(sv[u][rt][2], sv[u][rt][3])),
                             fmaxf(fmaxf(sv[u][rt][4], sv[u][rt][5]), fmaxf(sv[u][rt][6], sv[u][rt][7]))));
      }
      mx = max_x32(max_x16(mx));
      if (lg == 0) smax[w][rt * 16 + lr] = mx;
    }
    if (first) {
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int j = 0; j < MS; ++j) {
        const int key = (st0 + j) * 32 + 8 * lg;
        const int vo = (j < nst && key < nkeys) ? ((16 * w + lr) * a.cap + key) * 2 : vbytes;
        vf[j] = __builtin_amdgcn_raw_buffer_load_b128(vrs, vo, 0, 0);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
    lds_barrier();

    // ---- 2. probabilities against the block max, row sums
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
      const int rr = rt * 16 + lr;
      float M = smax[0][rr];
#pragma unroll
      for (int ww = 1; ww < NW; ++ww) M = fmaxf(M, smax[ww][rr]);
      const float mc = (M == -INFINITY ? 0.0f : M) * c;
      float ps = 0.0f;
#pragma unroll
      for (int u = 0; u < SW; ++u) {
        const int sl = w + NW * u;
        float pv[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          pv[j] = __builtin_amdgcn_exp2f(fmaf(sv[u][rt][j], c, -mc));  // exp2(-inf) = 0 when masked
          ps += pv[j];
        }
        uint32_t hi[4], lo[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          hi[e] = pack_bf16x2(pv[2 * e], pv[2 * e + 1]);
          // p - bf16(p) is exact in float32
          lo[e] = pack_bf16x2(pv[2 * e] - __uint_as_float(hi[e] << 16),
                              pv[2 * e + 1] - __uint_as_float(hi[e] & 0xffff0000u));
        }
        *(uint4 *)&sp[rr][32 * sl + 8 * lg] = make_uint4(hi[0], hi[1], hi[2], hi[3]);
        *(uint4 *)&spl[rr][32 * sl + 8 * lg] = make_uint4(lo[0], lo[1], lo[2], lo[3]);
      }
      ps = sum_x32(sum_x16(ps));
      if (lg == 0) ssum[w][rr] = ps;
    }
    lds_barrier();

    // ---- 3. O^T for dimensions 16 w .. 16 w + 15 over all of the keys
    f32x4 oacc[RT];
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) oacc[rt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int j = 0; j < MS; ++j) {
      if (j < nst) {
        i32x4 vv = vf[j];
        const int key = (st0 + j) * 32 + 8 * lg;
        if (key + 8 > nkeys) {  // slots never written for this step: zero
          const int valid = nkeys - key;
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const uint32_t lo = 2 * e < valid ? 0x0000ffffu : 0u;
            const uint32_t hi = 2 * e + 1 < valid ? 0xffff0000u : 0u;
            vv[e] &= (int)(lo | hi);
          }
        }
#pragma unroll
        for (int rt = 0; rt < RT; ++rt) {
          const uint4 pf = *(const uint4 *)&sp[rt * 16 + lr][32 * j + 8 * lg];
          const uint4 pl = *(const uint4 *)&spl[rt * 16 + lr][32 * j + 8 * lg];
          oacc[rt] = mfma16(__builtin_bit_cast(bf16x8, vv), as_bf16x8(pf), oacc[rt]);
          oacc[rt] = mfma16(__builtin_bit_cast(bf16x8, vv), as_bf16x8(pl), oacc[rt]);
        }
      }
    }
    // lane holds dimensions 16 w + 4 lg .. + 3 of row rb + 16 rt + lr
    const size_t base = ((size_t)g * a.n_chunks + split) * R;
#pragma unroll
    for (int rt = 0; rt < RT; ++rt) {
      const int r = rb + rt * 16 + lr;
      if (r < R) *(f32x4 *)&a.part_o[(base + r) * D + 16 * w + 4 * lg] = oacc[rt];
    }
    if (threadIdx.x < RB) {
      const int rr = threadIdx.x;
      const int r = rb + rr;
      if (r < R) {
        float M = smax[0][rr], L = ssum[0][rr];
#pragma unroll
        for (int ww = 1; ww < NW; ++ww) {
          M = fmaxf(M, smax[ww][rr]);
          L += ssum[ww][rr];
        }
        // row max in units of the scaled score (s * scale)
        *(float2 *)&a.part_ml[(base + r) * 2] = make_float2(M == -INFINITY ? M : M * a.scale, L);
      }
    }
    lds_barrier();  // sp, sq, sanc, smax, ssum free for the next row block
  };
  // the first block straight after the cache reads (no loop around it, so
  // the cache registers are not loop-carried and only the staging loads are
  // waited for before scoring starts)
  row_block(rb0, true);
  if constexpr (LOOP)
    for (int rb = RB; rb < R; rb += RB) {
      stage_loads(rb);
      row_block(rb, false);
    }
}

// Combines the key ranges of one (row t, query head) and writes the
// attention output in the packed operand layout of the O projection.  The
// 256 threads form 4 range groups x 64 column lanes.  The partial outputs of
// the first 4 ranges of every group are loaded together with the row
// statistics, before any wait (one memory round trip for up to 16 ranges);
// the range weights exp(m_c - M) go through LDS; the groups are added in LDS.
template <int D>
__global__ __launch_bounds__(256) void k_attn_merge(AttnArgs a, uint16_t *__restrict__ out, int ks) {
  constexpr int DPT = D / 64;  // columns per lane
  constexpr int MAXC = 512;
  constexpr int PK = 4;        // ranges per group loaded up front
  __shared__ float sw[MAXC];
  __shared__ float red[8];
  __shared__ float acc[4][D];
  const int t = blockIdx.x, head = blockIdx.y;
  const int G = a.n_heads / a.n_kv;
  const int g = head / G;
  const int R = a.n_tok * G;
  const int r = t * G + (head - g * G);
  const int nc = a.n_chunks;
  const int cg = threadIdx.x >> 6, lt = threadIdx.x & 63;
  const float2 *ml = (const float2 *)a.part_ml + (size_t)g * nc * R + r;
  const float *po = a.part_o + ((size_t)g * nc * R + r) * D + lt * DPT;
  const size_t cstride = (size_t)R * D;
  // ---- every load first: this thread's range statistics, its group's
  // first PK partial outputs
  float2 mlv = make_float2(-INFINITY, 0.0f);
  if ((int)threadIdx.x < nc) mlv = ml[(size_t)threadIdx.x * R];
  float v[PK][DPT];
#pragma unroll
  for (int k = 0; k < PK; ++k) {
    const int cc = cg + 4 * k;
#pragma unroll
    for (int e = 0; e < DPT; ++e) v[k][e] = cc < nc ? po[(size_t)cc * cstride + e] : 0.0f;
  }
  float m = mlv.x;
  for (int cc = threadIdx.x + 256; cc < nc; cc += 256) m = fmaxf(m, ml[(size_t)cc * R].x);
  for (int o = 32; o > 0; o >>= 1) m = fmaxf(m, __shfl_xor(m, o, 64));
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = m;
  __syncthreads();
  const float M = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
  float l = 0.0f;
  if ((int)threadIdx.x < nc) {
    const float wgt = mlv.x == -INFINITY ? 0.0f : expf(mlv.x - M);
    sw[threadIdx.x] = wgt;
    l = wgt * mlv.y;
  }
  for (int cc = threadIdx.x + 256; cc < nc; cc += 256) {
    const float2 x = ml[(size_t)cc * R];
    const float wgt = x.x == -INFINITY ? 0.0f : expf(x.x - M);
    sw[cc] = wgt;
    l += wgt * x.y;
  }
  for (int o = 32; o > 0; o >>= 1) l += __shfl_xor(l, o, 64);
  if ((threadIdx.x & 63) == 0) red[4 + (threadIdx.x >> 6)] = l;
  __syncthreads();
  const float L = red[4] + red[5] + red[6] + red[7];
  float o[DPT];
#pragma unroll
  for (int e = 0; e < DPT; ++e) o[e] = 0.0f;
#pragma unroll
  for (int k = 0; k < PK; ++k) {
    const int cc = cg + 4 * k;
    if (cc < nc)
#pragma unroll
      for (int e = 0; e < DPT; ++e) o[e] += sw[cc] * v[k][e];
  }
  for (int cc = cg + 4 * PK; cc < nc; cc += 4)
#pragma unroll
    for (int e = 0; e < DPT; ++e) o[e] += sw[cc] * po[(size_t)cc * cstride + e];

#pragma unroll
  for (int e = 0; e < DPT; ++e) acc[cg][lt * DPT + e] = o[e];
  __syncthreads();
  if (threadIdx.x < D / 8) {
    const int d0 = threadIdx.x * 8;
    const float inv = 1.0f / L;
    uint16_t b[8];
#pragma unroll
    for (int e = 0; e < 8; ++e)
      b[e] = f2bf((acc[0][d0 + e] + acc[1][d0 + e] + acc[2][d0 + e] + acc[3][d0 + e]) * inv);
    uint4 pk;
    pk.x = b[0] | ((uint32_t)b[1] << 16);
    pk.y = b[2] | ((uint32_t)b[3] << 16);
    pk.z = b[4] | ((uint32_t)b[5] << 16);
    pk.w = b[6] | ((uint32_t)b[7] << 16);
    *(uint4 *)(out + packed_index(t, head * D + d0, ks)) = pk;
  }
  // the last head also clears the padding columns of the packed row (the
  // GEMM reads K in whole chunks)
  const int width = a.n_heads * D;
  if (head == a.n_heads - 1) {
    for (int k0 = width + (int)threadIdx.x * 8; k0 < ks * 32; k0 += 256 * 8)
      *(uint4 *)(out + packed_index(t, k0, ks)) = make_uint4(0, 0, 0, 0);
  }
}

// Threads per workgroup of the register merge: one wave, so that the few
// thousand threads of a step spread over many compute units.
constexpr int kMergeThreads = 64;

// Merge for few key ranges (nc <= NCM): one thread per (row t, query head,
// 8 output dimensions).  Every load -- the range statistics and the 8
// dimensions of every range's partial output -- goes out before any use
// (one memory round trip); the thread writes its 8 dimensions as one
// 16-byte word of the packed operand layout of the O projection.
template <int D, int NCM>
__global__ __launch_bounds__(kMergeThreads) void k_attn_merge_reg(AttnArgs a,
                                                                  uint16_t *__restrict__ out, int ks) {
  constexpr int TPP = D / 8;  // threads per (row, head)
  const int nc = a.n_chunks;
  const int G = a.n_heads / a.n_kv;
  const int R = a.n_tok * G;
  // wave-uniform descriptors of the whole partial buffers; every load is
  // branch-free (ranges c >= nc and threads past the last (row, head) point
  // past the end and read zero)
  const int mbytes = __builtin_amdgcn_readfirstlane(a.n_kv * nc * R * 8);
  const int obytes = __builtin_amdgcn_readfirstlane(a.n_kv * nc * R * D * 4);
  const __amdgpu_buffer_rsrc_t mrs =
      __builtin_amdgcn_make_buffer_rsrc(uniform_ptr(a.part_ml), 0, mbytes, kBufferDword3);
  const __amdgpu_buffer_rsrc_t ors =
      __builtin_amdgcn_make_buffer_rsrc(uniform_ptr(a.part_o), 0, obytes, kBufferDword3);
  const int gid = blockIdx.x * kMergeThreads + threadIdx.x;
  const int pair = gid / TPP, part = gid - pair * TPP;
  const bool live = pair < a.n_tok * a.n_heads;
  const int t = pair / a.n_heads, head = pair - t * a.n_heads;
  const int g = head / G;
  const int r = t * G + (head - g * G);
  float2 st[NCM];
  f32x4 lo[NCM], hi[NCM];
#pragma unroll
  for (int c = 0; c < NCM; ++c) {
    const int row = (g * nc + c) * R + r;
    const bool in = live && c < nc;
    const int mo = in ? row * 8 : mbytes;
    const int oo = in ? (row * D + part * 8) * 4 : obytes;
    st[c].x = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(mrs, mo, 0, 0));
    st[c].y = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(mrs, mo + 4, 0, 0));
    lo[c] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(ors, oo, 0, 0));
    hi[c] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(ors, oo + 16, 0, 0));
  }
  __builtin_amdgcn_sched_barrier(0);  // all loads issued before any use
#pragma unroll
  for (int c = 0; c < NCM; ++c)
    if (c >= nc) st[c].x = -INFINITY;
  float M = st[0].x;
#pragma unroll
  for (int c = 1; c < NCM; ++c) M = fmaxf(M, st[c].x);
  float L = 0.0f;
  f32x4 o0 = {0.f, 0.f, 0.f, 0.f}, o1 = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int c = 0; c < NCM; ++c) {
    const float wgt = st[c].x == -INFINITY ? 0.0f : expf(st[c].x - M);
    L += wgt * st[c].y;
    o0 += wgt * lo[c];
    o1 += wgt * hi[c];
  }
  const float inv = 1.0f / L;
  uint4 pk;
  pk.x = f2bf(o0[0] * inv) | ((uint32_t)f2bf(o0[1] * inv) << 16);
  pk.y = f2bf(o0[2] * inv) | ((uint32_t)f2bf(o0[3] * inv) << 16);
  pk.z = f2bf(o1[0] * inv) | ((uint32_t)f2bf(o1[1] * inv) << 16);
  pk.w = f2bf(o1[2] * inv) | ((uint32_t)f2bf(o1[3] * inv) << 16);
  if (!live) return;
  *(uint4 *)(out + packed_index(t, head * D + part * 8, ks)) = pk;
  // the last head's threads clear the row's padding columns (the GEMM
  // reads K in whole chunks)
  if (head == a.n_heads - 1) {
    for (int k0 = a.n_heads * D + part * 8; k0 < ks * 32; k0 += TPP * 8)
      *(uint4 *)(out + packed_index(t, k0, ks)) = make_uint4(0, 0, 0, 0);
  }
}

}  // namespace

int attn_row_tiles(int rows) {
  // row blocks of at most kAttnMaxRowTiles tiles, as even as the tile count
  // allows
  const int tiles = (rows + 15) / 16;
  const int n_rb = (tiles + kAttnMaxRowTiles - 1) / kAttnMaxRowTiles;
  return (tiles + n_rb - 1) / n_rb;
}

bool attn_rb_split(int n_kv, int head_dim, int nkeys, int rows) {
  // a workgroup per row block while the launch stays within 16 rounds of
  // workgroups (the row blocks of one key range share its reads through
  // the XCD's L2); beyond that each workgroup walks its row blocks and
  // reads its keys once.  13B at prefix 8192: 65 rows 9.83 -> 9.35 ms per
  // step, 129 rows 13.57 -> 13.36 against a limit of 4 rounds.
  const int rt = attn_row_tiles(rows);
  const int n_rb = (rows + 16 * rt - 1) / (16 * rt);
  if (n_rb == 1) return true;
  const int steps = (nkeys + 31) / 32;
  const int ms2 = 2 * (head_dim / 16);
  return (long long)n_kv * n_rb * ((steps + ms2 - 1) / ms2) <= 16LL * kAttnCUs;
}

int attn_steps_per_wave(int n_kv, int head_dim, int nkeys, int rows) {
  // two steps per wave while the workgroups fit the compute units at one
  // each; beyond that one step, two workgroups per unit
  const int steps = (nkeys + 31) / 32;
  const int rt = attn_row_tiles(rows);
  const int n_rb = (rows + 16 * rt - 1) / (16 * rt);
  // a workgroup that walks several row blocks keeps its keys in registers
  // across them: two steps per wave (the one-step form spills there)
  if (n_rb > 1 && !attn_rb_split(n_kv, head_dim, nkeys, rows)) return 2;
  const int ms2 = 2 * (head_dim / 16);
  const long long units2 = (long long)n_kv * n_rb * ((steps + ms2 - 1) / ms2);
  return units2 > kAttnCUs ? 1 : 2;
}

int attn_splits(int n_kv, int head_dim, int nkeys, int rows) {
  // at most SW head_dim / 16 steps of 32 keys per workgroup, and about
  // kAttnTargetGroups workgroups in all (key ranges x row blocks) while
  // every one has kAttnMinSteps steps (shorter ranges cost more in partials
  // and merging than the extra workgroups gain)
  const int steps = (nkeys + 31) / 32;
  const int ms = attn_steps_per_wave(n_kv, head_dim, nkeys, rows) * (head_dim / 16);
  const int n_rb = attn_rb_split(n_kv, head_dim, nkeys, rows)
                       ? (rows + 16 * attn_row_tiles(rows) - 1) / (16 * attn_row_tiles(rows))
                       : 1;
  int sp = (steps + ms - 1) / ms;
  int fill = (kAttnTargetGroups + n_kv * n_rb - 1) / (n_kv * n_rb);
  const int most = (steps + kAttnMinSteps - 1) / kAttnMinSteps;
  if (fill > most) fill = most;
  if (sp < fill) sp = fill;
  return sp < 1 ? 1 : sp;
}

template <int D, int SW, bool LOOP>
hipError_t launch_attn_dsw(const AttnArgs &a, int rt, const dim3 &grid, hipStream_t s) {
  const dim3 block(D * 4);
  switch (rt) {
    case 1: hipLaunchKernelGGL((k_attn<D, 1, SW, LOOP>), grid, block, 0, s, a); break;
    case 2: hipLaunchKernelGGL((k_attn<D, 2, SW, LOOP>), grid, block, 0, s, a); break;
    case 3: hipLaunchKernelGGL((k_attn<D, 3, SW, LOOP>), grid, block, 0, s, a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <int D>
hipError_t launch_attn_d(const AttnArgs &a, hipStream_t s) {
  const int rows = a.n_tok * (a.n_heads / a.n_kv);
  const int nkeys = a.kv_len + a.n_tok;
  const int rt = attn_row_tiles(rows);
  const int n_rb = (rows + 16 * rt - 1) / (16 * rt);
  const bool loop = n_rb > 1 && !attn_rb_split(a.n_kv, D, nkeys, rows);
  const dim3 grid(a.n_kv * a.n_chunks * (loop ? 1 : n_rb));
  const bool one = attn_steps_per_wave(a.n_kv, D, nkeys, rows) == 1;
  if (loop)
    return one ? launch_attn_dsw<D, 1, true>(a, rt, grid, s) : launch_attn_dsw<D, 2, true>(a, rt, grid, s);
  return one ? launch_attn_dsw<D, 1, false>(a, rt, grid, s) : launch_attn_dsw<D, 2, false>(a, rt, grid, s);
}

hipError_t launch_attn_bf16(const AttnArgs &a, hipStream_t s) {
  if (a.n_chunks != attn_splits(a.n_kv, a.head_dim, a.kv_len + a.n_tok,
                                a.n_tok * (a.n_heads / a.n_kv)))
    return hipErrorInvalidValue;
  if (a.head_dim == 128) return launch_attn_d<128>(a, s);
  if (a.head_dim == 64) return launch_attn_d<64>(a, s);
  return hipErrorInvalidValue;
}

hipError_t launch_attn_merge_bf16(const AttnArgs &a, uint16_t *out_packed, int out_ks,
                                  hipStream_t s) {
  if (a.n_chunks > 512) return hipErrorInvalidValue;
  if (a.n_chunks <= 16 && (a.head_dim == 128 || a.head_dim == 64)) {
    const int threads = a.n_tok * a.n_heads * (a.head_dim / 8);
    const dim3 g((threads + kMergeThreads - 1) / kMergeThreads), b(kMergeThreads);
    if (a.head_dim == 128) {
      if (a.n_chunks <= 8)
        hipLaunchKernelGGL((k_attn_merge_reg<128, 8>), g, b, 0, s, a, out_packed, out_ks);
      else
        hipLaunchKernelGGL((k_attn_merge_reg<128, 16>), g, b, 0, s, a, out_packed, out_ks);
    } else {
      if (a.n_chunks <= 8)
        hipLaunchKernelGGL((k_attn_merge_reg<64, 8>), g, b, 0, s, a, out_packed, out_ks);
      else
        hipLaunchKernelGGL((k_attn_merge_reg<64, 16>), g, b, 0, s, a, out_packed, out_ks);
    }
    return hipGetLastError();
  }
  dim3 grid(a.n_tok, a.n_heads);
  if (a.head_dim == 128)
    hipLaunchKernelGGL(k_attn_merge<128>, grid, dim3(256), 0, s, a, out_packed, out_ks);
  else if (a.head_dim == 64)
    hipLaunchKernelGGL(k_attn_merge<64>, grid, dim3(256), 0, s, a, out_packed, out_ks);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace sb
