// Merge of partial attention results over key segments. Softmax over a union
// of key sets factors over the sets (contiguous key segments, one per
// worker, as in the segment-based sequence parallelism of paper Sec. I and II):
//
//     LSE_i = log sum_s exp(LSE_s,i),   O_i = sum_s exp(LSE_s,i - LSE_i) O_s,i
//
// computed here with the largest partial LSE subtracted first. Bound by HBM:
// each row reads P (d + 1) floats and writes d + 1. Thread t of the grid
// takes float4 t of the output (row t / (d/4), its d/4 float4 pieces in
// order), so a wave moves consecutive 16-byte pieces across row boundaries;
// the row width is a template parameter (TPR = d/4 pieces, d a multiple of 8
// up to 160), which keeps the division by it a multiply.
#include <math.h>

#include "vitattn_common.h"
#include "vitattn_launch.h"

namespace vitattn {

template <int TPR>
__global__ __launch_bounds__(256) void attn_merge_kernel(const float* __restrict__ o_parts,
                                                         const float* __restrict__ lse_parts, float* __restrict__ o,
                                                         float* __restrict__ lse, int P, long rows) {
  const long t = (long)blockIdx.x * 256 + threadIdx.x;
  const long row = t / TPR;
  const int c4 = (int)(t - row * TPR);
  if (row >= rows) return;
  // fmaxf ignores a NaN partial here; its weight below is NaN and poisons the row
  float m = -INFINITY;
  for (int p = 0; p < P; ++p) m = fmaxf(m, lse_parts[(size_t)p * rows + row]);
  float tot = 0.f;
  float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
  // partials in groups of four: the group's loads are issued before any is used
  constexpr int G = 4;
  int p0 = 0;
  for (; p0 + G <= P; p0 += G) {
    float4 x[G];
    float w[G];
#pragma unroll
    for (int u = 0; u < G; ++u) {
      const size_t pr = (size_t)(p0 + u) * rows + row;
      x[u] = reinterpret_cast<const float4*>(o_parts + pr * (4 * TPR))[c4];
      w[u] = lse_parts[pr];
    }
#pragma unroll
    for (int u = 0; u < G; ++u) {
      const float wu = expf(w[u] - m);
      tot += wu;
      acc.x += wu * x[u].x;
      acc.y += wu * x[u].y;
      acc.z += wu * x[u].z;
      acc.w += wu * x[u].w;
    }
  }
  for (int p = p0; p < P; ++p) {
    const size_t pr = (size_t)p * rows + row;
    const float w = expf(lse_parts[pr] - m);
    const float4 x = reinterpret_cast<const float4*>(o_parts + pr * (4 * TPR))[c4];
    tot += w;
    acc.x += w * x.x;
    acc.y += w * x.y;
    acc.z += w * x.z;
    acc.w += w * x.w;
  }
  const float inv = 1.f / tot;
  reinterpret_cast<float4*>(o + (size_t)row * (4 * TPR))[c4] =
      make_float4(acc.x * inv, acc.y * inv, acc.z * inv, acc.w * inv);
  if (c4 == 0) lse[row] = m + logf(tot);
}

template <int TPR>
static hipError_t merge_t(const MergeArgs& a) {
  const long rows = (long)a.BH * a.N;
  const long blocks = (rows * TPR + 255) / 256;
  hipLaunchKernelGGL(attn_merge_kernel<TPR>, dim3((unsigned)blocks), dim3(256), 0, a.stream, a.o_parts, a.lse_parts,
                     a.o, a.lse, a.P, rows);
  return hipGetLastError();
}

// d = 8 .. 160 in steps of 8: TPR = 2 .. 40 in steps of 2
template <int TPR>
static hipError_t merge_dispatch(const MergeArgs& a) {
  if constexpr (TPR > 40) {
    return hipErrorInvalidValue;
  } else {
    return a.d == 4 * TPR ? merge_t<TPR>(a) : merge_dispatch<TPR + 2>(a);
  }
}

hipError_t launch_merge(const MergeArgs& a) { return merge_dispatch<2>(a); }

}  // namespace vitattn
