// Merge of partial attention results over key segments. Softmax over a union
// of key sets factors over the sets (contiguous sequence segments, each GPU
// computing a partial self-attention for its segment: paper Sec. I and II):
//
//     LSE_i = log sum_s exp(LSE_s,i),   O_i = sum_s exp(LSE_s,i - LSE_i) O_s,i
//
// computed here with the largest partial LSE subtracted first. Bound by HBM:
// each row reads P (d + 1) floats and writes d + 1. One thread per four
// columns of a row; a block covers 256 / (d / 4) rows.
#include <math.h>

#include "vitattn_common.h"
#include "vitattn_launch.h"

namespace vitattn {

template <int D>
__global__ __launch_bounds__(256) void attn_merge_kernel(const float* __restrict__ o_parts,
                                                         const float* __restrict__ lse_parts, float* __restrict__ o,
                                                         float* __restrict__ lse, int P, long rows) {
  constexpr int TPR = D / 4;        // threads per row
  constexpr int RPB = 256 / TPR;    // rows per block
  const long row = (long)blockIdx.x * RPB + threadIdx.x / TPR;
  const int c4 = threadIdx.x % TPR;
  if (row >= rows) return;
  // fmaxf ignores a NaN partial here; its weight below is NaN and poisons the row
  float m = -INFINITY;
  for (int p = 0; p < P; ++p) m = fmaxf(m, lse_parts[(size_t)p * rows + row]);
  float tot = 0.f;
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  for (int p = 0; p < P; ++p) {
    const size_t pr = (size_t)p * rows + row;
    const float w = expf(lse_parts[pr] - m);
    const float4 x = reinterpret_cast<const float4*>(o_parts + pr * D)[c4];
    tot += w;
    acc.x += w * x.x;
    acc.y += w * x.y;
    acc.z += w * x.z;
    acc.w += w * x.w;
  }
  const float inv = 1.f / tot;
  reinterpret_cast<float4*>(o + (size_t)row * D)[c4] = make_float4(acc.x * inv, acc.y * inv, acc.z * inv, acc.w * inv);
  if (c4 == 0) lse[row] = m + logf(tot);
}

template __global__ void attn_merge_kernel<128>(const float* __restrict__, const float* __restrict__,
                                                float* __restrict__, float* __restrict__, int, long);
template __global__ void attn_merge_kernel<64>(const float* __restrict__, const float* __restrict__,
                                               float* __restrict__, float* __restrict__, int, long);

template <int D>
static hipError_t merge_d(const MergeArgs& a) {
  constexpr int RPB = 256 / (D / 4);
  const long rows = (long)a.BH * a.N;
  hipLaunchKernelGGL(attn_merge_kernel<D>, dim3((unsigned)((rows + RPB - 1) / RPB)), dim3(256), 0, a.stream,
                     a.o_parts, a.lse_parts, a.o, a.lse, a.P, rows);
  return hipGetLastError();
}

hipError_t launch_merge(const MergeArgs& a) { return a.d == 128 ? merge_d<128>(a) : merge_d<64>(a); }

}  // namespace vitattn
