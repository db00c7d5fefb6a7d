// bf16 forward kernels for gfx950 other than the GEMM: weight packing,
// embedding + tree metadata + RoPE table, and RMSNorm of the fp32 residual
// rows into the packed operand layout of the GEMM.
#include <math.h>

#include "sb_device.h"
#include "sb_internal_fwd.h"

namespace sb {
namespace {

// ---------------------------------------------------------------------------
// packing
// ---------------------------------------------------------------------------

struct PackArgs {
  const uint16_t *src0, *src1, *src2;
  uint16_t *dst;
  int kind;
  int K;        // source columns
  int ks;       // packed k-steps (K padded to whole 8-k-step chunks)
  int tiles;
  int n_heads, n_kv, head_dim, ffn, rows0;  // rows0: rows of src0 for O/DOWN/LM
};

// Source row of tile row r: returns the matrix and row, or nullptr.
__device__ const uint16_t *pack_src_row(const PackArgs &a, int tile, int r) {
  switch (a.kind) {
    case SB_W_QKV: {
      const int d = a.head_dim, ht = d / 16;
      const int qt = a.n_heads * ht, kt = a.n_kv * ht;
      if (tile < qt + kt) {
        const uint16_t *m = tile < qt ? a.src0 : a.src1;
        const int idx = tile < qt ? tile : tile - qt;
        const int head = idx / ht, u = idx % ht;
        const int dim = r < 8 ? 8 * u + r : d / 2 + 8 * u + (r - 8);
        return m + (size_t)(head * d + dim) * a.K;
      }
      const int idx = tile - qt - kt;
      const int row = idx * 16 + r;
      if (row >= a.n_kv * d) return nullptr;
      return a.src2 + (size_t)row * a.K;
    }
    case SB_W_GATE_UP: {
      const int f = tile * 8 + (r & 7);
      if (f >= a.ffn) return nullptr;
      return (r < 8 ? a.src0 : a.src1) + (size_t)f * a.K;
    }
    default: {
      const int row = tile * 16 + r;
      if (row >= a.rows0) return nullptr;
      return a.src0 + (size_t)row * a.K;
    }
  }
}

__global__ __launch_bounds__(256) void k_pack(PackArgs a) {
  const size_t total = (size_t)a.tiles * a.ks * 64;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
       i += (size_t)gridDim.x * blockDim.x) {
    const int lane = (int)(i & 63);
    const size_t ts = i >> 6;
    const int s = (int)(ts % a.ks);
    const int tile = (int)(ts / a.ks);
    const uint16_t *row = pack_src_row(a, tile, lane & 15);
    const int k0 = 32 * s + 8 * (lane >> 4);
    uint16_t v[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = (row && k0 + e < a.K) ? row[k0 + e] : (uint16_t)0;
    uint4 o;
    o.x = v[0] | ((uint32_t)v[1] << 16);
    o.y = v[2] | ((uint32_t)v[3] << 16);
    o.z = v[4] | ((uint32_t)v[5] << 16);
    o.w = v[6] | ((uint32_t)v[7] << 16);
    ((uint4 *)a.dst)[i] = o;
  }
}

// ---------------------------------------------------------------------------
// embedding + tree metadata + RoPE table
// ---------------------------------------------------------------------------

template <typename ET>
__device__ __forceinline__ float load_embed(const ET *e, size_t i);
template <>
__device__ __forceinline__ float load_embed<uint16_t>(const uint16_t *e, size_t i) {
  return bf2f(e[i]);
}
template <>
__device__ __forceinline__ float load_embed<float>(const float *e, size_t i) {
  return e[i];
}

template <typename ET>
__global__ __launch_bounds__(256) void k_embed_meta(EmbedArgs a, TreeArg tree) {
  const int t = blockIdx.x;
  float *h = a.h + (size_t)t * a.hidden;
  if (t < a.n_tok) {
    int tok = a.tokens[t];
    tok = tok < 0 ? 0 : (tok >= a.vocab ? a.vocab - 1 : tok);  // ids are clamped
    const ET *e = (const ET *)a.embed + (size_t)tok * a.hidden;
    if (sizeof(ET) == 2 && (a.hidden & 7) == 0) {
      // bf16 rows: 8 elements per 16-byte load, every load of the row issued
      // before the first store (hidden <= 16384: at most 8 per thread)
      constexpr int kMaxV = 8;
      uint4 v[kMaxV];
      const int nv = a.hidden >> 3;
#pragma unroll
      for (int j = 0; j < kMaxV; ++j) {
        const int i = threadIdx.x + j * 256;
        if (i < nv) v[j] = ((const uint4 *)e)[i];
      }
#pragma unroll
      for (int j = 0; j < kMaxV; ++j) {
        const int i = threadIdx.x + j * 256;
        if (i < nv) {
          const uint32_t w[4] = {v[j].x, v[j].y, v[j].z, v[j].w};
          float4 lo, hi;
          lo.x = bf2f((uint16_t)(w[0] & 0xffff)); lo.y = bf2f((uint16_t)(w[0] >> 16));
          lo.z = bf2f((uint16_t)(w[1] & 0xffff)); lo.w = bf2f((uint16_t)(w[1] >> 16));
          hi.x = bf2f((uint16_t)(w[2] & 0xffff)); hi.y = bf2f((uint16_t)(w[2] >> 16));
          hi.z = bf2f((uint16_t)(w[3] & 0xffff)); hi.w = bf2f((uint16_t)(w[3] >> 16));
          ((float4 *)h)[2 * i] = lo;
          ((float4 *)h)[2 * i + 1] = hi;
        }
      }
    } else {
      for (int k = threadIdx.x; k < a.hidden; k += blockDim.x) h[k] = load_embed<ET>(e, k);
    }
  } else {
    for (int k = threadIdx.x; k < a.hidden; k += blockDim.x) h[k] = 0.0f;
  }
  // this row's depth, position and ancestor mask, then its RoPE angles.
  // The tree (kernel arguments: a dynamically indexed read is a memory
  // access) goes to LDS in one parallel copy before the parent chase.
  __shared__ int s_pos;
  __shared__ int16_t s_par[SB_MAX_ROWS];
  for (int i = threadIdx.x; i < tree.n; i += blockDim.x) s_par[i] = tree.parent[i];
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t m[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    int depth = 0;
    if (t < tree.n) {
      int j = t;
      for (int guard = 0; guard < SB_MAX_ROWS && j >= 0; ++guard) {
#pragma unroll
        for (int w = 0; w < 8; ++w)
          if (w == (j >> 5)) m[w] |= 1u << (j & 31);
        j = s_par[j];
        if (j >= 0) ++depth;
      }
    }
    s_pos = a.kv_len + depth;
    a.meta->pos[t] = a.kv_len + depth;
#pragma unroll
    for (int w = 0; w < 8; ++w) a.meta->anc[t][w] = m[w];
  }
  __syncthreads();
  if (a.rope && t < a.n_tok) {
    const int half = a.head_dim / 2;
    for (int j = threadIdx.x; j < half; j += blockDim.x) {
      const double ang = (double)s_pos * a.theta[j];
      double sn, cs;
      sincos(ang, &sn, &cs);
      a.rope[t * half + j] = make_float2((float)cs, (float)sn);
    }
  }
}

// ---------------------------------------------------------------------------
// RMSNorm of the fp32 residual rows into the packed bf16 operand layout
// ---------------------------------------------------------------------------

// Threads per row of the RMSNorm kernel.
constexpr int kNormThreads = 512;

// One workgroup per row; a thread holds IPT groups of 8 columns in registers
// (one read of the row), the sum of squares is reduced across the block, and
// each group is written as one 16-byte store.
// With delta set, the n_delta slices of the previous projection (one per K
// range of a split-K GEMM, [n_delta][n_tok][hidden]) are first summed in
// slice order and added to the residual row, which is written back.
//
// The norm is applied in factored form, RMSNorm(h) g W^T = r (h g) W^T: the
// packed output is bf16(h g), and r = 1/sqrt(mean(h^2) + eps) goes to
// rs[t] for the projection's epilogue to multiply by.
//
// tap (H-RAD features, nullable): with tap_normed == 0 the residual row
// after the delta slices are added; with tap_normed != 0 the normalised row
// (h r) g in float32 (the last layer's state as the final norm leaves it).
//
// Every load of a thread (residual, all kMaxSplit delta slices, gains) is a
// buffer load issued before the first use, so a row costs one memory round
// trip; slices past n_delta, columns past hidden and rows past n_tok read
// zero (out-of-range offsets).
template <int IPT>
__global__ __launch_bounds__(kNormThreads) void k_rmsnorm_pack(float *__restrict__ h,
                                                               const float *__restrict__ delta,
                                                               int n_delta,
                                                               const float *__restrict__ g,
                                                               int hidden, int ks, int n_tok,
                                                               float eps,
                                                               uint16_t *__restrict__ out,
                                                               float *__restrict__ rs,
                                                               float *__restrict__ tap,
                                                               int tap_normed) {
  const int t = blockIdx.x;
  __shared__ float red[kNormThreads / 64];
  const int items = ks * 4;
  const bool live = t < n_tok;
  const int row_bytes = hidden * 4;
  const __amdgpu_buffer_rsrc_t hrs = __builtin_amdgcn_make_buffer_rsrc(
      (void *)(h + (size_t)(live ? t : 0) * hidden), 0, live ? row_bytes : 0, kBufferDword3);
  const int dbytes = delta ? n_delta * n_tok * row_bytes : 0;
  const __amdgpu_buffer_rsrc_t drs =
      __builtin_amdgcn_make_buffer_rsrc((void *)(delta ? delta : h), 0, dbytes, kBufferDword3);
  const __amdgpu_buffer_rsrc_t grs =
      __builtin_amdgcn_make_buffer_rsrc((void *)g, 0, row_bytes, kBufferDword3);
  f32x4 hv[IPT][2], dv[IPT][kMaxSplit][2], gv[IPT][2];
#pragma unroll
  for (int j = 0; j < IPT; ++j) {
    const int k0 = (threadIdx.x + j * kNormThreads) * 8;
    const int vo = k0 < hidden ? k0 * 4 : row_bytes;
#pragma unroll
    for (int hh = 0; hh < 2; ++hh) {
      hv[j][hh] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(hrs, vo, hh * 16, 0));
      gv[j][hh] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(grs, vo, hh * 16, 0));
    }
#pragma unroll
    for (int sl = 0; sl < kMaxSplit; ++sl) {
      const int dvo = (k0 < hidden && live) ? ((sl * n_tok + t) * hidden + k0) * 4 : dbytes;
#pragma unroll
      for (int hh = 0; hh < 2; ++hh)
        dv[j][sl][hh] =
            __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(drs, dvo, hh * 16, 0));
    }
  }
  float ss = 0.0f;
#pragma unroll
  for (int j = 0; j < IPT; ++j) {
    const int k0 = (threadIdx.x + j * kNormThreads) * 8;
    if (delta) {  // residual add of the previous projection, slices in order
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) {
        f32x4 d = dv[j][0][hh];
#pragma unroll
        for (int sl = 1; sl < kMaxSplit; ++sl) d += dv[j][sl][hh];  // missing slices read 0
        hv[j][hh] += d;
      }
      if (live && k0 < hidden) {
        f32x4 *dst = (f32x4 *)(h + (size_t)t * hidden + k0);
        dst[0] = hv[j][0];
        dst[1] = hv[j][1];
        if (tap && !tap_normed) {  // the residual after the previous layer, for H-RAD
          f32x4 *tp = (f32x4 *)(tap + (size_t)t * hidden + k0);
          tp[0] = hv[j][0];
          tp[1] = hv[j][1];
        }
      }
    }
#pragma unroll
    for (int hh = 0; hh < 2; ++hh)
#pragma unroll
      for (int e = 0; e < 4; ++e) ss += hv[j][hh][e] * hv[j][hh][e];
  }
  for (int o = 32; o > 0; o >>= 1) ss += __shfl_xor(ss, o, 64);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
  __syncthreads();
  ss = red[0];
#pragma unroll
  for (int i = 1; i < kNormThreads / 64; ++i) ss += red[i];
  const float scale = live ? 1.0f / sqrtf(ss / (float)hidden + eps) : 0.0f;
  if (rs && threadIdx.x == 0) rs[t] = scale;  // padding rows get 0
#pragma unroll
  for (int j = 0; j < IPT; ++j) {
    const int it = threadIdx.x + j * kNormThreads;
    if (it >= items) continue;
    const int k0 = it * 8;
    // columns past hidden have zero residual and gain: they pack to zero
    uint16_t v[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = f2bf(hv[j][e >> 2][e & 3] * gv[j][e >> 2][e & 3]);
    uint4 o;
    o.x = v[0] | ((uint32_t)v[1] << 16);
    o.y = v[2] | ((uint32_t)v[3] << 16);
    o.z = v[4] | ((uint32_t)v[5] << 16);
    o.w = v[6] | ((uint32_t)v[7] << 16);
    *(uint4 *)(out + packed_index(t, k0, ks)) = o;
    if (tap && tap_normed && live && k0 < hidden) {  // the final norm's output, float32
      f32x4 *tp = (f32x4 *)(tap + (size_t)t * hidden + k0);
      tp[0] = (hv[j][0] * scale) * gv[j][0];
      tp[1] = (hv[j][1] * scale) * gv[j][1];
    }
  }
}

}  // namespace

hipError_t launch_pack_bf16(int kind, const sb_model_config &c, const void *src0, const void *src1,
                            const void *src2, void *dst, hipStream_t s) {
  PackArgs a;
  a.src0 = (const uint16_t *)src0;
  a.src1 = (const uint16_t *)src1;
  a.src2 = (const uint16_t *)src2;
  a.dst = (uint16_t *)dst;
  a.kind = kind;
  a.n_heads = c.n_heads;
  a.n_kv = c.n_kv_heads;
  a.head_dim = c.head_dim;
  a.ffn = c.ffn;
  const PackGeom g = pack_geom(c, kind);
  a.K = g.K;
  a.ks = g.ks;
  a.tiles = g.tiles;
  a.rows0 = g.rows;
  const size_t total = (size_t)a.tiles * a.ks * 64;
  size_t blocks = (total + 255) / 256;
  if (blocks > 65536) blocks = 65536;
  hipLaunchKernelGGL(k_pack, dim3((unsigned)blocks), dim3(256), 0, s, a);
  return hipGetLastError();
}

hipError_t launch_embed_meta(const EmbedArgs &a, const TreeArg &tree, int blocks, int bf16,
                             hipStream_t s) {
  if (bf16)
    hipLaunchKernelGGL(k_embed_meta<uint16_t>, dim3(blocks), dim3(256), 0, s, a, tree);
  else
    hipLaunchKernelGGL(k_embed_meta<float>, dim3(blocks), dim3(256), 0, s, a, tree);
  return hipGetLastError();
}

hipError_t launch_rmsnorm_pack(float *h, const float *delta, int n_delta, const float *g,
                               int hidden, int ks, int n_tok, int n_pad, float eps, uint16_t *out,
                               float *rs, hipStream_t s, float *tap, int tap_normed) {
  if (hidden % 8 != 0 || n_delta < 1 || n_delta > kMaxSplit) return hipErrorInvalidValue;
  const int ipt = (ks * 4 + kNormThreads - 1) / kNormThreads;
  switch (ipt) {
#define SB_IPT(n)                                                                              \
  case n:                                                                                      \
    hipLaunchKernelGGL(k_rmsnorm_pack<n>, dim3(n_pad), dim3(kNormThreads), 0, s, h, delta,        \
                       n_delta, g, hidden, ks, n_tok, eps, out, rs, tap, tap_normed);          \
    break;
    SB_IPT(1) SB_IPT(2) SB_IPT(3) SB_IPT(4) SB_IPT(5) SB_IPT(6) SB_IPT(7) SB_IPT(8)
#undef SB_IPT
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace sb
