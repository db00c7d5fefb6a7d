// H-RAD's draft-length predictor (Section "H-RAD", equations for z_t and
// s_t): the features are the target's residual stream after each of its
// last K layers at the last accepted row, concatenated with the embedding
// of the new token; a 256/64/3 ReLU MLP maps them to three logits, and the
// class is their argmax (softmax is monotone).  float32 arithmetic.
#include "sb_device.h"
#include "sb_internal_fwd.h"

namespace sb {
namespace {

constexpr int kL1Threads = 256;

// The row and token the features come from: the last row of the walk's
// path and its next token; false when the result names no usable pair.
__device__ __forceinline__ bool hrad_source(const HradArgs &a, int *row, int *tok) {
  const int plen = a.res->path_len;
  if (plen < 1 || plen > SB_MAX_ROWS) return false;
  const int r = a.res->path[plen - 1];
  const int y = a.res->next_token;
  if (r < 0 || r >= a.max_rows || y < 0 || y >= a.vocab) return false;
  *row = r;
  *tok = y;
  return true;
}

// One workgroup per unit j of the first layer: y1[j] = ReLU(W1[j] . z + b1[j]),
// z = (tap 0 .. tap k-1 of the row, the token's embedding); a thread takes 4
// consecutive inputs per step (hidden is a multiple of 8, so 4 never straddle
// two parts of z).
__global__ __launch_bounds__(kL1Threads) void k_hrad_l1(HradArgs a) {
  __shared__ float red[kL1Threads / 64];
  const int j = blockIdx.x;
  int r = 0, y = 0;
  const bool ok = hrad_source(a, &r, &y);
  const int H = a.hidden;
  const int din = (a.k + 1) * H;
  const float *wr = a.w1 + (size_t)j * din;
  float acc = 0.0f;
  if (ok) {
    for (int i = threadIdx.x * 4; i < din; i += kL1Threads * 4) {
      const f32x4 wv = *(const f32x4 *)(wr + i);
      const int k = i / H, d = i - k * H;
      f32x4 zv;
      if (k < a.k) {
        zv = *(const f32x4 *)(a.taps + ((size_t)k * a.max_rows + r) * H + d);
      } else {
        const uint2 e = *(const uint2 *)(a.embed + (size_t)y * H + d);
        zv = f32x4{bf2f((uint16_t)(e.x & 0xffff)), bf2f((uint16_t)(e.x >> 16)),
                   bf2f((uint16_t)(e.y & 0xffff)), bf2f((uint16_t)(e.y >> 16))};
      }
#pragma unroll
      for (int c = 0; c < 4; ++c) acc += wv[c] * zv[c];
    }
  }
  for (int o = 32; o > 0; o >>= 1) acc += __shfl_xor(acc, o, 64);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = acc;
  __syncthreads();
  if (threadIdx.x == 0) {
    float sum = red[0];
#pragma unroll
    for (int w = 1; w < kL1Threads / 64; ++w) sum += red[w];
    a.y1[j] = ok ? fmaxf(sum + a.b1[j], 0.0f) : 0.0f;
  }
}

// The 64-unit layer (thread m computes unit m), then the 3 logits and their
// argmax (lowest index on ties) by thread 0.
__global__ __launch_bounds__(SB_HRAD_H2) void k_hrad_tail(HradArgs a) {
  __shared__ float y1[SB_HRAD_H1], y2[SB_HRAD_H2];
  int r = 0, y = 0;
  const bool ok = hrad_source(a, &r, &y);
  for (int i = threadIdx.x; i < SB_HRAD_H1; i += SB_HRAD_H2) y1[i] = a.y1[i];
  __syncthreads();
  {
    const int m = threadIdx.x;
    const float *w = a.w2 + (size_t)m * SB_HRAD_H1;
    float acc = 0.0f;
    for (int i = 0; i < SB_HRAD_H1; ++i) acc += w[i] * y1[i];
    y2[m] = fmaxf(acc + a.b2[m], 0.0f);
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    float lg[SB_HRAD_CLASSES];
    int best = 0;
    for (int c = 0; c < SB_HRAD_CLASSES; ++c) {
      const float *w = a.w3 + (size_t)c * SB_HRAD_H2;
      float acc = 0.0f;
      for (int i = 0; i < SB_HRAD_H2; ++i) acc += w[i] * y2[i];
      lg[c] = acc + a.b3[c];
      if (c > 0 && lg[c] > lg[best]) best = c;
    }
    for (int c = 0; c < SB_HRAD_CLASSES; ++c) a.logits3[c] = ok ? lg[c] : 0.0f;
    *a.cls = ok ? best : -1;
  }
}

}  // namespace

hipError_t launch_hrad(const HradArgs &a, hipStream_t s) {
  if (a.hidden % 8 != 0 || a.k < 1) return hipErrorInvalidValue;
  hipLaunchKernelGGL(k_hrad_l1, dim3(SB_HRAD_H1), dim3(kL1Threads), 0, s, a);
  hipLaunchKernelGGL(k_hrad_tail, dim3(1), dim3(SB_HRAD_H2), 0, s, a);
  return hipGetLastError();
}

}  // namespace sb
