// float32 forward kernels.  The float32 models are the small exactness and
// parity shapes; these kernels favour a plain, deterministic structure over
// speed (one wavefront per output dot product, one workgroup per attention
// row), while following the same tree semantics as the bf16 path.
#include <math.h>

#include "sb_device.h"
#include "sb_internal_fwd.h"

namespace sb {
namespace {

__device__ __forceinline__ float wave_sumf(float v) {
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

__global__ __launch_bounds__(256) void k_f32_rmsnorm(const float *__restrict__ h,
                                                     const float *__restrict__ g, int hidden,
                                                     float eps, float *__restrict__ out) {
  const int t = blockIdx.x;
  __shared__ float red[4];
  const float *x = h + (size_t)t * hidden;
  float ss = 0.0f;
  for (int k = threadIdx.x; k < hidden; k += 256) ss += x[k] * x[k];
  ss = wave_sumf(ss);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
  __syncthreads();
  ss = red[0] + red[1] + red[2] + red[3];
  const float scale = 1.0f / sqrtf(ss / (float)hidden + eps);
  for (int k = threadIdx.x; k < hidden; k += 256) out[(size_t)t * hidden + k] = (x[k] * scale) * g[k];
}

// Y[t][m] (+)= sum_k X[t][k] W[m][k]; one wavefront per output.
__global__ __launch_bounds__(256) void k_f32_gemm(const float *__restrict__ X,
                                                  const float *__restrict__ W,
                                                  float *__restrict__ Y, int M, int K, int ldy,
                                                  int accumulate) {
  const int t = blockIdx.y;
  const int m = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (m >= M) return;
  const float *x = X + (size_t)t * K;
  const float *wr = W + (size_t)m * K;
  float s = 0.0f;
  for (int k = lane; k < K; k += 64) s += x[k] * wr[k];
  s = wave_sumf(s);
  if (lane == 0) {
    float *y = Y + (size_t)t * ldy + m;
    *y = accumulate ? *y + s : s;
  }
}

// q, k rotated at pos(t); k and v stored in cache slot kv_len + t.
__global__ __launch_bounds__(128) void k_f32_rope_qkv(const float *__restrict__ qkv, int n_heads,
                                                      int n_kv, int d,
                                                      const float2 *__restrict__ rope,
                                                      float *__restrict__ q, float *__restrict__ kc,
                                                      float *__restrict__ vc, int cap,
                                                      int kv_len) {
  const int t = blockIdx.x, hh = blockIdx.y;  // hh < n_heads + 2 * n_kv
  const int width = (n_heads + 2 * n_kv) * d;
  const float *row = qkv + (size_t)t * width + (size_t)hh * d;
  const int half = d / 2;
  for (int j = threadIdx.x; j < d; j += blockDim.x) {
    if (hh < n_heads + n_kv) {
      if (j >= half) continue;
      const float2 cs = rope[t * half + j];
      const float x1 = row[j], x2 = row[j + half];
      const float o1 = x1 * cs.x - x2 * cs.y;
      const float o2 = x2 * cs.x + x1 * cs.y;
      float *dst = hh < n_heads ? q + ((size_t)t * n_heads + hh) * d
                                : kc + ((size_t)(hh - n_heads) * cap + kv_len + t) * d;
      dst[j] = o1;
      dst[j + half] = o2;
    } else {
      const int g = hh - n_heads - n_kv;
      vc[((size_t)g * d + j) * cap + kv_len + t] = row[j];  // V cached transposed
    }
  }
}

// One workgroup per (row t, query head): scores of every visible key in
// LDS, softmax, weighted sum of V.
__global__ __launch_bounds__(256) void k_f32_attn(AttnArgs a, float *__restrict__ out) {
  extern __shared__ float sc[];  // [kv_len + n_tok]
  __shared__ float red[8];
  const int t = blockIdx.x, head = blockIdx.y;
  const int d = a.head_dim;
  const int G = a.n_heads / a.n_kv;
  const int g = head / G;
  const int nkeys = a.kv_len + a.n_tok;
  const float *qr = (const float *)a.q + ((size_t)t * a.n_heads + head) * d;
  const float *kc = (const float *)a.kc + (size_t)g * a.cap * d;
  const float *vt = (const float *)a.vc + (size_t)g * d * a.cap;  // [d][slot]
  float m = -INFINITY;
  for (int j = threadIdx.x; j < nkeys; j += 256) {
    bool ok = j < a.kv_len;
    if (!ok) {
      const int jj = j - a.kv_len;
      ok = (a.meta->anc[t][jj >> 5] >> (jj & 31)) & 1u;
    }
    float s = -INFINITY;
    if (ok) {
      float acc = 0.0f;
      for (int k = 0; k < d; ++k) acc += qr[k] * kc[(size_t)j * d + k];
      s = acc * a.scale;
    }
    sc[j] = s;
    m = fmaxf(m, s);
  }
  for (int o = 32; o > 0; o >>= 1) m = fmaxf(m, __shfl_xor(m, o, 64));
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = m;
  __syncthreads();
  m = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
  __syncthreads();
  float l = 0.0f;
  for (int j = threadIdx.x; j < nkeys; j += 256) {
    const float e = expf(sc[j] - m);
    sc[j] = e;
    l += e;
  }
  l = wave_sumf(l);
  if ((threadIdx.x & 63) == 0) red[4 + (threadIdx.x >> 6)] = l;
  __syncthreads();
  l = red[4] + red[5] + red[6] + red[7];
  for (int dd = threadIdx.x; dd < d; dd += 256) {
    float o = 0.0f;
    const float *vrow = vt + (size_t)dd * a.cap;
    for (int j = 0; j < nkeys; ++j) o += sc[j] * vrow[j];
    out[(size_t)t * a.n_heads * d + (size_t)head * d + dd] = o / l;
  }
}

__global__ __launch_bounds__(256) void k_f32_swiglu(const float *__restrict__ gu, int ffn,
                                                    float *__restrict__ act) {
  const int t = blockIdx.y;
  const int f = blockIdx.x * 256 + threadIdx.x;
  if (f >= ffn) return;
  const float gv = gu[(size_t)t * 2 * ffn + f];
  const float uv = gu[(size_t)t * 2 * ffn + ffn + f];
  act[(size_t)t * ffn + f] = gv / (1.0f + expf(-gv)) * uv;
}

}  // namespace

hipError_t launch_f32_rmsnorm(const float *h, const float *g, int hidden, int n_tok, float eps,
                              float *out, hipStream_t s) {
  hipLaunchKernelGGL(k_f32_rmsnorm, dim3(n_tok), dim3(256), 0, s, h, g, hidden, eps, out);
  return hipGetLastError();
}

hipError_t launch_f32_gemm(const float *X, const float *W, float *Y, int n_tok, int M, int K,
                           int ldy, int accumulate, hipStream_t s) {
  dim3 grid((M + 3) / 4, n_tok);
  hipLaunchKernelGGL(k_f32_gemm, grid, dim3(256), 0, s, X, W, Y, M, K, ldy, accumulate);
  return hipGetLastError();
}

hipError_t launch_f32_rope_qkv(const float *qkv, const sb_model_config &c, int n_tok,
                               const float2 *rope, float *q, float *kc, float *vc, int cap,
                               int kv_len, hipStream_t s) {
  dim3 grid(n_tok, c.n_heads + 2 * c.n_kv_heads);
  hipLaunchKernelGGL(k_f32_rope_qkv, grid, dim3(128), 0, s, qkv, c.n_heads, c.n_kv_heads,
                     c.head_dim, rope, q, kc, vc, cap, kv_len);
  return hipGetLastError();
}

hipError_t launch_f32_attn(const AttnArgs &a, float *out, hipStream_t s) {
  const size_t lds = (size_t)(a.kv_len + a.n_tok) * sizeof(float);
  dim3 grid(a.n_tok, a.n_heads);
  hipLaunchKernelGGL(k_f32_attn, grid, dim3(256), lds, s, a, out);
  return hipGetLastError();
}

hipError_t launch_f32_swiglu(const float *gu, int n_tok, int ffn, float *act, hipStream_t s) {
  dim3 grid((ffn + 255) / 256, n_tok);
  hipLaunchKernelGGL(k_f32_swiglu, grid, dim3(256), 0, s, gu, ffn, act);
  return hipGetLastError();
}

}  // namespace sb
