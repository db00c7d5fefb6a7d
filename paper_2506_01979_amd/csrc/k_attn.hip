// Branch-masked attention over a shared prefix KV cache (bf16, matrix cores).
//
// Every tree row attends to the committed prefix (cache slots [0, kv_len))
// and to the tree rows on its own path root..i (slots kv_len + j with bit j
// of its ancestor mask) -- the branch-causal mask under which one forward
// scores all branches at once while each branch sees exactly what a separate
// causal forward of that branch would see (Section "Branch Resampling").
//
// Work split: one workgroup per (KV head, chunk of 128 key slots) over the
// combined key range [0, kv_len + n_tok).  The V cache is stored transposed
// ([d][slot]), so both matrix-core operands that come from the cache -- K
// rows for S^T = K Q^T and V^T rows for O^T = V^T P^T -- are 16-byte runs of
// consecutive elements read straight from HBM.  Every cache load of the
// chunk is issued before the first wait, so a workgroup pays one memory
// latency; a prefix tile is fetched once and reused by every branch and
// every query head of the KV group (GQA).  Queries and probabilities go
// through LDS.  The workgroup writes an unnormalised partial (row max m, row
// sum l, sum p v) per query row; the merge kernel combines the chunks with
// the log-sum-exp rule.
#include <math.h>

#include "sb_device.h"
#include "sb_internal_fwd.h"

namespace sb {
namespace {

constexpr int CH = kAttnChunk;  // keys per workgroup
constexpr int RB = 64;          // query rows per block (4 row tiles)
constexpr int PAD = 8;          // LDS row padding (bf16 elements)

// 8 consecutive bf16 of a V^T row starting at slot `key`; slots >= nkeys
// (never written for this step) read as zero, and nothing past the cache
// capacity is touched.
__device__ __forceinline__ uint4 load_vt8(const uint16_t *row, int key, int nkeys, int cap) {
  if (key + 8 <= nkeys) return *(const uint4 *)(row + key);
  uint4 v = make_uint4(0, 0, 0, 0);
  if (key < nkeys && key + 8 <= cap) {
    v = *(const uint4 *)(row + key);
    const int keep = nkeys - key;  // 1..7 valid elements
    uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int e = 0; e < 8; ++e)
      if (e >= keep) w[e >> 1] &= (e & 1) ? 0x0000ffffu : 0xffff0000u;
    v = make_uint4(w[0], w[1], w[2], w[3]);
  }
  return v;
}

template <int D>
__global__ __launch_bounds__(256) void k_attn(AttnArgs a) {
  constexpr int KSD = D / 32;    // k-steps over head_dim
  constexpr int DT = D / 16;     // d tiles
  constexpr int DTW = DT / 4;    // d tiles per wave (4 waves)
  constexpr int VV = D / 8;      // 16-byte vectors per query row
  constexpr int KK = CH / 32;    // k-steps over the chunk's keys
  __shared__ uint16_t P[RB][CH + PAD];  // probabilities (bf16), row-major
  __shared__ uint16_t Qs[RB][D + PAD];  // query rows of this block
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
  const uint16_t *__restrict__ vt = (const uint16_t *)a.vc + (size_t)g * D * a.cap;
  const uint16_t *__restrict__ q = (const uint16_t *)a.q;

  // ---- every cache load of the chunk, issued up front
  uint4 ka[2][KSD];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int slot = key0 + (2 * w + i) * 16 + lr;
#pragma unroll
    for (int s = 0; s < KSD; ++s)
      ka[i][s] = slot < nkeys ? *(const uint4 *)(kc + (size_t)slot * D + 32 * s + 8 * lg)
                              : make_uint4(0, 0, 0, 0);
  }
  uint4 va[DTW][KK];
#pragma unroll
  for (int i = 0; i < DTW; ++i) {
    const uint16_t *row = vt + (size_t)((w * DTW + i) * 16 + lr) * a.cap;
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) va[i][kk] = load_vt8(row, key0 + kk * 32 + 8 * lg, nkeys, a.cap);
  }

  for (int r0 = 0; r0 < R; r0 += RB) {
    // stage the query rows of this block
    for (int idx = threadIdx.x; idx < RB * VV; idx += 256) {
      const int rr = idx / VV, dv = (idx % VV) * 8;
      const int r = r0 + rr;
      uint4 v = make_uint4(0, 0, 0, 0);
      if (r < R) {
        const int t = r / G, hl = r - t * G;
        v = *(const uint4 *)(q + ((size_t)t * a.n_heads + g * G + hl) * D + dv);
      }
      *(uint4 *)&Qs[rr][dv] = v;
    }
    __syncthreads();
    // ---- S^T = K Q^T for this wave's 2 key tiles x 4 row tiles
    f32x4 sacc[2][4];
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int rt = 0; rt < 4; ++rt) sacc[i][rt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < KSD; ++s) {
#pragma unroll
      for (int rt = 0; rt < 4; ++rt) {
        const uint4 qb = *(const uint4 *)&Qs[rt * 16 + lr][32 * s + 8 * lg];
#pragma unroll
        for (int i = 0; i < 2; ++i)
          sacc[i][rt] = mfma16(as_bf16x8(ka[i][s]), as_bf16x8(qb), sacc[i][rt]);
      }
    }
    // ---- scale, mask, row max over this wave's 32 keys
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
      if (lg == 0) redm[w][rt * 16 + lr] = m;
    }
    __syncthreads();
    float lsum[4];
#pragma unroll
    for (int rt = 0; rt < 4; ++rt) {
      const int rr = rt * 16 + lr;
      const float m = fmaxf(fmaxf(redm[0][rr], redm[1][rr]), fmaxf(redm[2][rr], redm[3][rr]));
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
    }
#pragma unroll
    for (int rt = 0; rt < 4; ++rt)
      if (lg == 0) redl[w][rt * 16 + lr] = lsum[rt];
    __syncthreads();  // P and redl complete
    // ---- O^T = V^T P^T for this wave's d tiles
    f32x4 oacc[DTW][4];
#pragma unroll
    for (int i = 0; i < DTW; ++i)
#pragma unroll
      for (int rt = 0; rt < 4; ++rt) oacc[i][rt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
      uint4 pbv[4];
#pragma unroll
      for (int rt = 0; rt < 4; ++rt) pbv[rt] = *(const uint4 *)&P[rt * 16 + lr][kk * 32 + 8 * lg];
#pragma unroll
      for (int i = 0; i < DTW; ++i)
#pragma unroll
        for (int rt = 0; rt < 4; ++rt)
          oacc[i][rt] = mfma16(as_bf16x8(va[i][kk]), as_bf16x8(pbv[rt]), oacc[i][rt]);
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
    if (threadIdx.x < RB) {
      const int rr = threadIdx.x;
      const int r = r0 + rr;
      if (r < R) {
        const float m = fmaxf(fmaxf(redm[0][rr], redm[1][rr]), fmaxf(redm[2][rr], redm[3][rr]));
        const float l = redl[0][rr] + redl[1][rr] + redl[2][rr] + redl[3][rr];
        *(float2 *)&a.part_ml[(base + r) * 2] = make_float2(m, l);
      }
    }
    __syncthreads();  // Qs, P, redm, redl free for the next row block
  }
}

// Combines the chunks of one (row t, query head) and writes the attention
// output in the packed operand layout of the O projection.  The 256 threads
// form 4 chunk groups x 64 column lanes: the chunk weights exp(m_c - M) are
// computed once into LDS, each group sums its chunks with independent loads,
// and the groups are added in LDS.
template <int D>
__global__ __launch_bounds__(256) void k_attn_merge(AttnArgs a, uint16_t *__restrict__ out, int ks) {
  constexpr int DPT = D / 64;  // columns per lane
  constexpr int MAXC = 512;
  __shared__ float sw[MAXC];
  __shared__ float red[8];
  __shared__ float acc[4][D];
  const int t = blockIdx.x, head = blockIdx.y;
  const int G = a.n_heads / a.n_kv;
  const int g = head / G;
  const int R = a.n_tok * G;
  const int r = t * G + (head - g * G);
  const int nc = a.n_chunks;
  const float2 *ml = (const float2 *)a.part_ml + (size_t)g * nc * R + r;
  float m = -INFINITY;
  for (int cc = threadIdx.x; cc < nc; cc += 256) {
    const float mv = ml[(size_t)cc * R].x;
    sw[cc] = mv;
    m = fmaxf(m, mv);
  }
  for (int o = 32; o > 0; o >>= 1) m = fmaxf(m, __shfl_xor(m, o, 64));
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = m;
  __syncthreads();
  const float M = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
  float l = 0.0f;
  for (int cc = threadIdx.x; cc < nc; cc += 256) {
    const float mv = sw[cc];
    const float wgt = mv == -INFINITY ? 0.0f : expf(mv - M);
    sw[cc] = wgt;
    l += wgt * ml[(size_t)cc * R].y;
  }
  for (int o = 32; o > 0; o >>= 1) l += __shfl_xor(l, o, 64);
  if ((threadIdx.x & 63) == 0) red[4 + (threadIdx.x >> 6)] = l;
  __syncthreads();
  const float L = red[4] + red[5] + red[6] + red[7];
  const int cg = threadIdx.x >> 6, lt = threadIdx.x & 63;
  float o[DPT];
#pragma unroll
  for (int e = 0; e < DPT; ++e) o[e] = 0.0f;
  const float *po = a.part_o + ((size_t)g * nc * R + r) * D + lt * DPT;
  const size_t cstride = (size_t)R * D;
  int cc = cg;
  for (; cc + 12 < nc; cc += 16) {  // four chunks of this group per batch
    float v[4][DPT];
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int e = 0; e < DPT; ++e) v[j][e] = po[(size_t)(cc + 4 * j) * cstride + e];
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int e = 0; e < DPT; ++e) o[e] += sw[cc + 4 * j] * v[j][e];
  }
  for (; cc < nc; cc += 4)
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
  if (a.n_chunks > 512) return hipErrorInvalidValue;
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
