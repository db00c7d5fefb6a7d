// Branch-masked attention over a shared prefix KV cache (bf16, matrix cores).
//
// Every tree row attends to the committed prefix (cache slots [0, kv_len))
// and to the tree rows on its own path root..i (slots kv_len + j with bit j
// of its ancestor mask) -- the branch-causal mask under which one forward
// scores all branches at once while each branch sees exactly what a separate
// causal forward of that branch would see (Section "Branch Resampling").
//
// Work split: one workgroup per (KV head, chunk of 128 key slots) over the
// combined key range [0, kv_len + n_tok).  The chunk's V is staged in LDS
// once (transposed for the P.V operand) and its K is read once per
// 64-query-row block, so a prefix tile is fetched from HBM once and reused by
// every branch and every query head of the KV group (GQA).  The workgroup
// writes an unnormalised partial (row max m, row sum l, sum p v) per query
// row; a merge kernel combines the chunks with the usual log-sum-exp rule.
#include <math.h>

#include "sb_device.h"
#include "sb_internal_fwd.h"

namespace sb {
namespace {

constexpr int CH = kAttnChunk;  // keys per workgroup
constexpr int RB = 64;          // query rows per block (4 row tiles)
constexpr int VPAD = 8;         // LDS row padding (bf16 elements)

template <int D>
__global__ __launch_bounds__(256) void k_attn(AttnArgs a) {
  constexpr int KSD = D / 32;           // k-steps over head_dim
  constexpr int DT = D / 16;            // d tiles
  constexpr int DTW = DT / 4;           // d tiles per wave (4 waves)
  __shared__ uint16_t Vt[D][CH + VPAD];  // V chunk, transposed
  __shared__ uint16_t P[RB][CH + VPAD];  // probabilities (bf16)
  __shared__ float redm[4][RB];
  __shared__ float redl[4][RB];

  const int g = blockIdx.x, c = blockIdx.y;
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int lr = lane & 15, lg = lane >> 4;
  const int G = a.n_heads / a.n_kv;
  const int R = a.n_tok * G;
  const int key0 = c * CH;
  const int nkeys = a.kv_len + a.n_tok;
  const uint16_t *__restrict__ kc = (const uint16_t *)a.kc + (size_t)g * a.cap * D;
  const uint16_t *__restrict__ vc = (const uint16_t *)a.vc + (size_t)g * a.cap * D;
  const uint16_t *__restrict__ q = (const uint16_t *)a.q;

  // stage V^T for this chunk
  for (int idx = threadIdx.x; idx < CH * (D / 8); idx += 256) {
    const int key = idx / (D / 8);
    const int dv = (idx % (D / 8)) * 8;
    const int slot = key0 + key;
    uint4 v = make_uint4(0, 0, 0, 0);
    if (slot < nkeys) v = *(const uint4 *)(vc + (size_t)slot * D + dv);
    const uint32_t wv[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      Vt[dv + 2 * e][key] = (uint16_t)(wv[e] & 0xffff);
      Vt[dv + 2 * e + 1][key] = (uint16_t)(wv[e] >> 16);
    }
  }

  for (int r0 = 0; r0 < R; r0 += RB) {
    __syncthreads();  // Vt ready / P free
    // ---- S^T = K Q^T for this wave's 2 key tiles x 4 row tiles
    f32x4 sacc[2][4];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int rt = 0; rt < 4; ++rt) sacc[i][rt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < KSD; ++s) {
      uint4 ka[2], qb[4];
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        const int slot = key0 + (2 * w + i) * 16 + lr;
        ka[i] = slot < nkeys ? *(const uint4 *)(kc + (size_t)slot * D + 32 * s + 8 * lg)
                             : make_uint4(0, 0, 0, 0);
      }
#pragma unroll
      for (int rt = 0; rt < 4; ++rt) {
        const int r = r0 + rt * 16 + lr;
        if (r < R) {
          const int t = r / G, hl = r - t * G;
          qb[rt] = *(const uint4 *)(q + ((size_t)t * a.n_heads + g * G + hl) * D + 32 * s + 8 * lg);
        } else {
          qb[rt] = make_uint4(0, 0, 0, 0);
        }
      }
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int rt = 0; rt < 4; ++rt) sacc[i][rt] = mfma16(as_bf16x8(ka[i]), as_bf16x8(qb[rt]), sacc[i][rt]);
    }
    // ---- scale, mask, row max over this wave's 32 keys
    float mrow[4];
#pragma unroll
    for (int rt = 0; rt < 4; ++rt) {
      const int r = r0 + rt * 16 + lr;
      const int t = r < R ? r / G : 0;
      float m = -INFINITY;
#pragma unroll
      for (int i = 0; i < 2; ++i) {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int slot = key0 + (2 * w + i) * 16 + 4 * lg + e;
          bool ok = slot < a.kv_len;
          if (!ok && slot < nkeys) {
            const int j = slot - a.kv_len;
            ok = (a.meta->anc[t][j >> 5] >> (j & 31)) & 1u;
          }
          const float sv = ok ? sacc[i][rt][e] * a.scale : -INFINITY;
          sacc[i][rt][e] = sv;
          m = fmaxf(m, sv);
        }
      }
      m = fmaxf(m, __shfl_xor(m, 16, 64));
      m = fmaxf(m, __shfl_xor(m, 32, 64));
      mrow[rt] = m;
      if (lg == 0) redm[w][rt * 16 + lr] = m;
    }
    __syncthreads();
    float lsum[4];
#pragma unroll
    for (int rt = 0; rt < 4; ++rt) {
      const int rr = rt * 16 + lr;
      float m = fmaxf(fmaxf(redm[0][rr], redm[1][rr]), fmaxf(redm[2][rr], redm[3][rr]));
      const float mref = (m == -INFINITY) ? 0.0f : m;
      float l = 0.0f;
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        uint16_t pb[4];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float pv = expf(sacc[i][rt][e] - mref);  // exp(-inf) = 0 for masked keys
          l += pv;
          pb[e] = f2bf(pv);
        }
        uint2 st;
        st.x = pb[0] | ((uint32_t)pb[1] << 16);
        st.y = pb[2] | ((uint32_t)pb[3] << 16);
        *(uint2 *)&P[rr][(2 * w + i) * 16 + 4 * lg] = st;
      }
      l += __shfl_xor(l, 16, 64);
      l += __shfl_xor(l, 32, 64);
      lsum[rt] = l;
      mrow[rt] = m;
    }
    __syncthreads();  // all of P written, redm read
#pragma unroll
    for (int rt = 0; rt < 4; ++rt)
      if (lg == 0) redl[w][rt * 16 + lr] = lsum[rt];
    // ---- O^T = V^T P^T for this wave's d tiles
    f32x4 oacc[DTW][4];
#pragma unroll
    for (int i = 0; i < DTW; ++i)
#pragma unroll
      for (int rt = 0; rt < 4; ++rt) oacc[i][rt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kk = 0; kk < CH / 32; ++kk) {
      uint4 va[DTW], pbv[4];
#pragma unroll
      for (int i = 0; i < DTW; ++i) va[i] = *(const uint4 *)&Vt[(w * DTW + i) * 16 + lr][kk * 32 + 8 * lg];
#pragma unroll
      for (int rt = 0; rt < 4; ++rt) pbv[rt] = *(const uint4 *)&P[rt * 16 + lr][kk * 32 + 8 * lg];
#pragma unroll
      for (int i = 0; i < DTW; ++i)
#pragma unroll
        for (int rt = 0; rt < 4; ++rt) oacc[i][rt] = mfma16(as_bf16x8(va[i]), as_bf16x8(pbv[rt]), oacc[i][rt]);
    }
    const size_t base = ((size_t)g * a.n_chunks + c) * R;
#pragma unroll
    for (int i = 0; i < DTW; ++i) {
#pragma unroll
      for (int rt = 0; rt < 4; ++rt) {
        const int r = r0 + rt * 16 + lr;
        if (r < R) {
          const int d0 = (w * DTW + i) * 16 + 4 * lg;
          *(f32x4 *)&a.part_o[(base + r) * D + d0] = oacc[i][rt];
        }
      }
    }
    __syncthreads();  // redl written
    if (threadIdx.x < RB) {
      const int rr = threadIdx.x;
      const int r = r0 + rr;
      if (r < R) {
        const float m = fmaxf(fmaxf(redm[0][rr], redm[1][rr]), fmaxf(redm[2][rr], redm[3][rr]));
        const float l = redl[0][rr] + redl[1][rr] + redl[2][rr] + redl[3][rr];
        a.part_ml[(base + r) * 2 + 0] = m;
        a.part_ml[(base + r) * 2 + 1] = l;
      }
    }
  }
}

// Combines the chunks of one (row, head) and writes the attention output in
// the packed operand layout of the O projection.
template <int D>
__global__ __launch_bounds__(D) void k_attn_merge(AttnArgs a, uint16_t *__restrict__ out, int ks) {
  const int t = blockIdx.x, head = blockIdx.y;
  const int G = a.n_heads / a.n_kv;
  const int g = head / G;
  const int R = a.n_tok * G;
  const int r = t * G + (head - g * G);
  const int dd = threadIdx.x;
  float M = -INFINITY;
  for (int c = 0; c < a.n_chunks; ++c)
    M = fmaxf(M, a.part_ml[(((size_t)g * a.n_chunks + c) * R + r) * 2]);
  float L = 0.0f, o = 0.0f;
  for (int c = 0; c < a.n_chunks; ++c) {
    const size_t b = ((size_t)g * a.n_chunks + c) * R + r;
    const float m = a.part_ml[b * 2];
    if (m == -INFINITY) continue;
    const float wgt = expf(m - M);
    L += a.part_ml[b * 2 + 1] * wgt;
    o += a.part_o[b * D + dd] * wgt;
  }
  out[packed_index(t, head * D + dd, ks)] = f2bf(o / L);
}

}  // namespace

hipError_t launch_attn_bf16(const AttnArgs &a, hipStream_t s) {
  dim3 grid(a.n_kv, a.n_chunks);
  if (a.head_dim == 128)
    hipLaunchKernelGGL(k_attn<128>, grid, dim3(256), 0, s, a);
  else if (a.head_dim == 64)
    hipLaunchKernelGGL(k_attn<64>, grid, dim3(256), 0, s, a);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

hipError_t launch_attn_merge_bf16(const AttnArgs &a, uint16_t *out_packed, int out_ks,
                                  hipStream_t s) {
  dim3 grid(a.n_tok, a.n_heads);
  if (a.head_dim == 128)
    hipLaunchKernelGGL(k_attn_merge<128>, grid, dim3(128), 0, s, a, out_packed, out_ks);
  else if (a.head_dim == 64)
    hipLaunchKernelGGL(k_attn_merge<64>, grid, dim3(64), 0, s, a, out_packed, out_ks);
  else
    return hipErrorInvalidValue;
  return hipGetLastError();
}

}  // namespace sb
