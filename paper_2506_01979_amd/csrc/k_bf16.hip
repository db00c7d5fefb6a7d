// bf16 forward kernels for gfx950: weight packing, embedding + tree
// metadata, RMSNorm into the packed operand layout, and the skinny
// matrix-core GEMM with fused epilogues (RoPE + KV write, residual add,
// SwiGLU, logits).
//
// The verify forward multiplies n_rows (5..256) activation rows by every
// weight matrix once; the weights (13-140 GB) dominate the bytes, so the
// GEMM streams each weight tile from HBM exactly once with 16-byte loads in
// the operand order of v_mfma_f32_16x16x32_bf16 (the layout sb_pack_weight
// writes), keeps all activation rows of the step resident as B operands, and
// splits K across the 8 waves of a workgroup, reducing in LDS.  A workgroup
// owns one 16-row output tile, so every output element is finished inside one
// workgroup and its epilogue runs there.
#include <math.h>

#include "sb_device.h"
#include "sb_internal_fwd.h"

namespace sb {
namespace {

constexpr int kGemmThreads = 512;
constexpr int kGemmWaves = kGemmThreads / 64;

// ---------------------------------------------------------------------------
// packing
// ---------------------------------------------------------------------------

struct PackArgs {
  const uint16_t *src0, *src1, *src2;
  uint16_t *dst;
  int kind;
  int K;        // source columns
  int ks;       // packed k-steps (K padded to 32)
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
    const ET *e = (const ET *)a.embed;
    for (int k = threadIdx.x; k < a.hidden; k += blockDim.x)
      h[k] = load_embed<ET>(e, (size_t)tok * a.hidden + k);
  } else {
    for (int k = threadIdx.x; k < a.hidden; k += blockDim.x) h[k] = 0.0f;
  }
  // this row's depth, position and ancestor mask, then its RoPE angles
  __shared__ int s_pos;
  if (threadIdx.x == 0) {
    uint32_t m[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    int depth = 0;
    if (t < tree.n) {
      int j = t;
      for (int guard = 0; guard < SB_MAX_ROWS && j >= 0; ++guard) {
        m[j >> 5] |= 1u << (j & 31);
        j = tree.parent[j];
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

// One workgroup per row; a thread holds IPT groups of 8 columns in registers
// (one read of the row), the sum of squares is reduced across the block, and
// each group is written as one 16-byte store.
template <int IPT>
__global__ __launch_bounds__(256) void k_rmsnorm_pack(const float *__restrict__ h,
                                                      const float *__restrict__ g, int hidden,
                                                      int ks, int n_tok, float eps,
                                                      uint16_t *__restrict__ out) {
  const int t = blockIdx.x;
  __shared__ float red[4];
  const int items = ks * 4;
  float x[IPT][8];
  float ss = 0.0f;
  const bool live = t < n_tok;
#pragma unroll
  for (int j = 0; j < IPT; ++j) {
    const int it = threadIdx.x + j * 256;
    const int k0 = it * 8;
    if (live && it < items && k0 < hidden) {
      const float4 *src = (const float4 *)(h + (size_t)t * hidden + k0);
      const float4 p0 = src[0], p1 = src[1];
      x[j][0] = p0.x; x[j][1] = p0.y; x[j][2] = p0.z; x[j][3] = p0.w;
      x[j][4] = p1.x; x[j][5] = p1.y; x[j][6] = p1.z; x[j][7] = p1.w;
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) x[j][e] = 0.0f;
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) ss += x[j][e] * x[j][e];
  }
  for (int o = 32; o > 0; o >>= 1) ss += __shfl_xor(ss, o, 64);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
  __syncthreads();
  ss = red[0] + red[1] + red[2] + red[3];
  const float scale = live ? 1.0f / sqrtf(ss / (float)hidden + eps) : 0.0f;
#pragma unroll
  for (int j = 0; j < IPT; ++j) {
    const int it = threadIdx.x + j * 256;
    if (it >= items) continue;
    const int k0 = it * 8;
    uint16_t v[8];
    if (k0 < hidden) {
      const float4 g0 = *(const float4 *)(g + k0), g1 = *(const float4 *)(g + k0 + 4);
      const float gg[8] = {g0.x, g0.y, g0.z, g0.w, g1.x, g1.y, g1.z, g1.w};
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] = f2bf((x[j][e] * scale) * gg[e]);
    } else {
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] = 0;
    }
    uint4 o;
    o.x = v[0] | ((uint32_t)v[1] << 16);
    o.y = v[2] | ((uint32_t)v[3] << 16);
    o.z = v[4] | ((uint32_t)v[5] << 16);
    o.w = v[6] | ((uint32_t)v[7] << 16);
    *(uint4 *)(out + packed_index(t, k0, ks)) = o;
  }
}

// ---------------------------------------------------------------------------
// skinny matrix-core GEMM with fused epilogues
// ---------------------------------------------------------------------------

__device__ __forceinline__ void rope_pair(float x1, float x2, float2 cs, float *o1, float *o2) {
  *o1 = x1 * cs.x - x2 * cs.y;
  *o2 = x2 * cs.x + x1 * cs.y;
}

// Epilogue of one finished output pair: rows p and p + 8 of tile `tile`,
// activation row t, values v1 / v2.
template <int EPI>
__device__ __forceinline__ void epilogue(const GemmArgs &a, int tile, int p, int t, float v1,
                                         float v2) {
  if constexpr (EPI == EPI_QKV) {
    if (t >= a.n_tok) return;
    const int d = a.head_dim, ht = d / 16;
    const int qt = a.n_heads * ht, kt = a.n_kv * ht;
    if (tile < qt + kt) {
      const bool isq = tile < qt;
      const int idx = isq ? tile : tile - qt;
      const int head = idx / ht, u = idx % ht;
      const int j = 8 * u + p;
      float o1, o2;
      rope_pair(v1, v2, a.rope[t * (d / 2) + j], &o1, &o2);
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
  } else if constexpr (EPI == EPI_RESID) {
    if (t >= a.n_tok) return;
    const int d1 = tile * 16 + p, d2 = d1 + 8;
    float *hrow = a.h + (size_t)t * a.out_rows;
    if (d1 < a.out_rows) hrow[d1] += v1;
    if (d2 < a.out_rows) hrow[d2] += v2;
  } else if constexpr (EPI == EPI_SWIGLU) {
    const int f = tile * 8 + p;
    const float gsil = v1 / (1.0f + expf(-v1));
    a.act[packed_index(t, f, a.act_ks)] = f2bf(gsil * v2);
  } else {  // EPI_LOGITS
    if (t >= a.n_tok) return;
    const int v1i = tile * 16 + p, v2i = v1i + 8;
    float *lrow = a.logits + (size_t)t * a.out_rows;
    if (v1i < a.out_rows) lrow[v1i] = v1;
    if (v2i < a.out_rows) lrow[v2i] = v2;
  }
}

// A workgroup owns RT consecutive 16-row tiles; its 8 waves split K.  Each
// wave streams its weight fragments with a two-deep software pipeline
// (batch i+1 in flight while batch i feeds the matrix cores).
template <int TT, int EPI, int RT>
__global__ __launch_bounds__(kGemmThreads) void k_gemm(GemmArgs a) {
  extern __shared__ float red[];  // [waves][RT][TT][64 lanes][4]
  constexpr int U = TT <= 4 ? 2 : 1;
  const int tile0 = blockIdx.x * RT;
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int ks = a.ks;
  const int s0 = (ks * w) / kGemmWaves, s1 = (ks * (w + 1)) / kGemmWaves;
  const uint4 *Wt[RT];
#pragma unroll
  for (int r = 0; r < RT; ++r)
    Wt[r] = (const uint4 *)a.W + (size_t)min(tile0 + r, a.tiles - 1) * ks * 64 + lane;
  const uint4 *__restrict__ Xp = (const uint4 *)a.X + lane;

  bool tv[TT];
#pragma unroll
  for (int tt = 0; tt < TT; ++tt) tv[tt] = (tt * 16 + (lane & 15)) < a.n_tok;

  f32x4 acc[RT][TT];
#pragma unroll
  for (int r = 0; r < RT; ++r)
#pragma unroll
    for (int tt = 0; tt < TT; ++tt) acc[r][tt] = f32x4{0.f, 0.f, 0.f, 0.f};

  auto load = [&](int s, uint4(&av)[U][RT], uint4(&bv)[U][TT]) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
#pragma unroll
      for (int r = 0; r < RT; ++r)
        av[u][r] = (s + u < s1) ? load_stream(Wt[r] + (size_t)(s + u) * 64) : make_uint4(0, 0, 0, 0);
#pragma unroll
      for (int tt = 0; tt < TT; ++tt)
        bv[u][tt] = (s + u < s1 && tv[tt]) ? Xp[((size_t)tt * ks + s + u) * 64]
                                            : make_uint4(0, 0, 0, 0);
    }
  };
  auto compute = [&](uint4(&av)[U][RT], uint4(&bv)[U][TT]) {
#pragma unroll
    for (int u = 0; u < U; ++u)
#pragma unroll
      for (int r = 0; r < RT; ++r)
#pragma unroll
        for (int tt = 0; tt < TT; ++tt)
          acc[r][tt] = mfma16(as_bf16x8(av[u][r]), as_bf16x8(bv[u][tt]), acc[r][tt]);
  };
  if constexpr (TT <= 8) {
    uint4 a0[U][RT], b0[U][TT], a1[U][RT], b1[U][TT];
    int s = s0;
    if (s < s1) load(s, a0, b0);
    while (s < s1) {
      if (s + U < s1) load(s + U, a1, b1);
      compute(a0, b0);
      s += U;
      if (s >= s1) break;
      if (s + U < s1) load(s + U, a0, b0);
      compute(a1, b1);
      s += U;
    }
  } else {  // very wide trees: one batch at a time keeps the registers in budget
    for (int s = s0; s < s1; s += U) {
      uint4 a0[U][RT], b0[U][TT];
      load(s, a0, b0);
      compute(a0, b0);
    }
  }

#pragma unroll
  for (int r = 0; r < RT; ++r)
#pragma unroll
    for (int tt = 0; tt < TT; ++tt)
      *(f32x4 *)&red[((((size_t)w * RT + r) * TT + tt) * 64 + lane) * 4] = acc[r][tt];
  __syncthreads();

  // item = (tile r, pair p of rows p / p+8, token t)
  const int items = RT * 8 * 16 * TT;
  for (int it = threadIdx.x; it < items; it += kGemmThreads) {
    const int r = it / (128 * TT);
    const int rem = it - r * 128 * TT;
    const int p = rem & 7;
    const int t = rem >> 3;
    const int tt = t >> 4;
    const int l1 = (t & 15) + 16 * (p >> 2), e1 = p & 3;
    const int l2 = (t & 15) + 16 * ((p + 8) >> 2), e2 = (p + 8) & 3;
    float v1 = 0.f, v2 = 0.f;
#pragma unroll
    for (int ww = 0; ww < kGemmWaves; ++ww) {
      v1 += red[((((size_t)ww * RT + r) * TT + tt) * 64 + l1) * 4 + e1];
      v2 += red[((((size_t)ww * RT + r) * TT + tt) * 64 + l2) * 4 + e2];
    }
    if (tile0 + r < a.tiles) epilogue<EPI>(a, tile0 + r, p, t, v1, v2);
  }
}

template <int TT, int EPI, int RT>
hipError_t launch_gemm_rt(const GemmArgs &a, hipStream_t s) {
  const size_t lds = (size_t)kGemmWaves * RT * TT * 64 * 4 * sizeof(float);
  static bool attr_set = false;
  if (!attr_set) {
    hipError_t e = hipFuncSetAttribute((const void *)k_gemm<TT, EPI, RT>,
                                       hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
    attr_set = true;
  }
  const int grid = (a.tiles + RT - 1) / RT;
  hipLaunchKernelGGL((k_gemm<TT, EPI, RT>), dim3(grid), dim3(kGemmThreads), lds, s, a);
  return hipGetLastError();
}

// Row tiles per workgroup: more tiles share the activation fragments (fewer
// bytes from L2 per weight byte) but leave fewer workgroups; measured best
// on MI355X for 33-row steps: 4 for >= 768 tiles (QKV, LM head), 2 for the
// gate/up GEMM, 1 for the 256-tile O and down GEMMs.
template <int TT, int EPI>
hipError_t launch_gemm_tt(const GemmArgs &a, hipStream_t s) {
  if constexpr (TT <= 3) {
    if (a.tiles >= 1700 || (a.tiles >= 700 && a.tiles < 1000)) return launch_gemm_rt<TT, EPI, 4>(a, s);
  }
  if constexpr (TT <= 4) {
    if (a.tiles >= 700) return launch_gemm_rt<TT, EPI, 2>(a, s);
  }
  return launch_gemm_rt<TT, EPI, 1>(a, s);
}

template <int EPI>
hipError_t launch_gemm_epi(const GemmArgs &a, int tt, hipStream_t s) {
  switch (tt) {
#define SB_TT(n) \
  case n:        \
    return launch_gemm_tt<n, EPI>(a, s);
    SB_TT(1) SB_TT(2) SB_TT(3) SB_TT(4) SB_TT(5) SB_TT(6) SB_TT(7) SB_TT(8)
    SB_TT(9) SB_TT(10) SB_TT(11) SB_TT(12) SB_TT(13) SB_TT(14) SB_TT(15) SB_TT(16)
#undef SB_TT
    default:
      return hipErrorInvalidValue;
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

hipError_t launch_rmsnorm_pack(const float *h, const float *g, int hidden, int ks, int n_tok,
                               int n_pad, float eps, uint16_t *out, hipStream_t s) {
  const int ipt = (ks * 4 + 255) / 256;
  switch (ipt) {
#define SB_IPT(n)                                                                              \
  case n:                                                                                      \
    hipLaunchKernelGGL(k_rmsnorm_pack<n>, dim3(n_pad), dim3(256), 0, s, h, g, hidden, ks, n_tok, \
                       eps, out);                                                              \
    break;
    SB_IPT(1) SB_IPT(2) SB_IPT(3) SB_IPT(4) SB_IPT(5) SB_IPT(6) SB_IPT(7) SB_IPT(8)
#undef SB_IPT
    default:
      return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_gemm(int epi, const GemmArgs &a, int tiles, int tt, hipStream_t s) {
  GemmArgs b = a;
  b.tiles = tiles;
  switch (epi) {
    case EPI_QKV:
      return launch_gemm_epi<EPI_QKV>(b, tt, s);
    case EPI_RESID:
      return launch_gemm_epi<EPI_RESID>(b, tt, s);
    case EPI_SWIGLU:
      return launch_gemm_epi<EPI_SWIGLU>(b, tt, s);
    case EPI_LOGITS:
      return launch_gemm_epi<EPI_LOGITS>(b, tt, s);
    default:
      return hipErrorInvalidValue;
  }
}

}  // namespace sb
