// Channel aggregation by attention with a learnable query (the Agg-Ch-ViT
// layer, paper Sec. II "Patch Embedding and Sequence Length"): per patch
// position m and head h, one query q_h shared by every patch attends over
// the C channel tokens of that patch:
//
//   s_c = scale q_h . k_mhc,  LSE = log sum_c exp(s_c),  o_mh = sum_c exp(s_c - LSE) v_mhc
//
// and the backward pass (dq_h sums over all patches, as q is shared):
//
//   dp_c = do . v_c,  D = do . o,  ds_c = p_c (dp_c - D),
//   dk_c = scale ds_c q_h,  dv_c = p_c do,  dq_h = scale sum_m sum_c ds_c k_c
//
// Many tiny attentions, bound by HBM bandwidth: one wave per (m, h). A
// [C][d] block is read (and dK, dV are written) as consecutive 1 KB chunks
// of 512 / d rows: lane l holds 8 columns, 8 (l % (d/8)) onward, of row
// l / (d/8) of the chunk, so every load and store instruction of the wave
// moves one contiguous piece. A row's dot products are the lane's 8 products
// summed over its d/8 lanes by an exchange butterfly (every lane of the row
// ends with the same, bitwise equal value); weighted sums over rows stay
// per lane and are summed across a chunk's rows once, at the end. A wave
// issues the loads of several chunks before using any of them.
// dq is reduced without atomics: each block sums a fixed range of patches
// into a partial in the workspace, then one pass adds the partials in a fixed
// order, so results are bitwise reproducible.
#include <math.h>

#include "vitattn_common.h"
#include "vitattn_launch.h"

namespace vitattn {

namespace {

__device__ __forceinline__ float wave_max(float x) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x = fmaxf(x, __shfl_xor(x, o));
  return x;
}

__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x += __shfl_xor(x, o);
  return x;
}

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// 8 bf16 values (one 16-byte piece) widened to fp32
__device__ __forceinline__ void widen8(const uint4 w, float (&x)[8]) {
  x[0] = bf16_lo(w.x);
  x[1] = bf16_hi(w.x);
  x[2] = bf16_lo(w.y);
  x[3] = bf16_hi(w.y);
  x[4] = bf16_lo(w.z);
  x[5] = bf16_hi(w.z);
  x[6] = bf16_lo(w.w);
  x[7] = bf16_hi(w.w);
}

// this lane's share of a dot product: 8 products accumulated in column order
__device__ __forceinline__ float dot8(const float (&a)[8], const float (&b)[8]) {
  float acc = 0.f;
#pragma unroll
  for (int e = 0; e < 8; ++e) acc = fmaf(a[e], b[e], acc);
  return acc;
}

// sum over the LPR lanes that hold one row (an aligned group of lanes); the
// pairwise adds are commutative, so every lane of the group gets the same bits
template <int LPR>
__device__ __forceinline__ float row_sum(float x) {
#pragma unroll
  for (int o = 1; o < LPR; o <<= 1) x += __shfl_xor(x, o);
  return x;
}

// sum of each of the lane's 8 values over the 64 / LPR rows of a chunk
// (lanes l, l + LPR, l + 2 LPR, ...); every such lane gets the same bits
template <int LPR>
__device__ __forceinline__ void chunk_rows_sum(float (&x)[8]) {
#pragma unroll
  for (int o = LPR; o < 64; o <<= 1)
#pragma unroll
    for (int e = 0; e < 8; ++e) x[e] += __shfl_xor(x[e], o);
}

__device__ __forceinline__ uint4 load16(const uint16_t* p) { return *reinterpret_cast<const uint4*>(p); }

__device__ __forceinline__ void store8(float* p, const float (&x)[8]) {
  reinterpret_cast<float4*>(p)[0] = make_float4(x[0], x[1], x[2], x[3]);
  reinterpret_cast<float4*>(p)[1] = make_float4(x[4], x[5], x[6], x[7]);
}

}  // namespace

template <int D>
__global__ __launch_bounds__(256) void attn_agg_fwd_kernel(const uint16_t* __restrict__ q,
                                                           const uint16_t* __restrict__ k,
                                                           const uint16_t* __restrict__ v, float* __restrict__ o,
                                                           float* __restrict__ lse, int MH, int H, int C, float c2) {
  constexpr int LPR = D / 8, RPC = 64 / LPR, G = kAggChunkGroup;
  const int wave = threadIdx.x >> 6;
  const int inst = blockIdx.x * 4 + wave;
  if (inst >= MH) return;  // whole waves exit together; no block barrier follows
  const int lane = threadIdx.x & 63;
  const int r = lane / LPR, cg = lane % LPR;  // row within a chunk, column group
  const int h = inst % H;
  float qv[8];
  widen8(load16(q + (size_t)h * D + cg * 8), qv);
  // this lane's piece of chunk 0 (chunk t is 512 elements further on)
  const uint16_t* kb = k + (size_t)inst * C * D + lane * 8;
  const uint16_t* vb = v + (size_t)inst * C * D + lane * 8;
  const int n_chunks = (C + RPC - 1) / RPC;

  float m_run = -INFINITY, l = 0.f;  // log2 units
  float acc[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) acc[e] = 0.f;
  for (int t0 = 0; t0 < n_chunks; t0 += G) {
    uint4 kr[G], vr[G];
    bool ok[G];
#pragma unroll
    for (int u = 0; u < G; ++u) {
      ok[u] = (t0 + u) * RPC + r < C;
      kr[u] = ok[u] ? load16(kb + (size_t)(t0 + u) * 512) : make_uint4(0u, 0u, 0u, 0u);
    }
#pragma unroll
    for (int u = 0; u < G; ++u) vr[u] = ok[u] ? load16(vb + (size_t)(t0 + u) * 512) : make_uint4(0u, 0u, 0u, 0u);
    float s[G], mx = -INFINITY;
#pragma unroll
    for (int u = 0; u < G; ++u) {
      float kx[8];
      widen8(kr[u], kx);
      s[u] = ok[u] ? row_sum<LPR>(dot8(kx, qv)) * c2 : -INFINITY;
      mx = fmaxf(mx, s[u]);
    }
    const float m_new = fmaxf(m_run, wave_max(mx));  // finite: every group holds a row
    const float alpha = exp2f(m_run - m_new);
    float ps = 0.f;
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] *= alpha;
#pragma unroll
    for (int u = 0; u < G; ++u) {
      const float p = ok[u] ? exp2f(s[u] - m_new) : 0.f;
      if (cg == 0) ps += p;  // one lane per row adds to the sum
      float vx[8];
      widen8(vr[u], vx);
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[e] = fmaf(p, vx[e], acc[e]);
    }
    l = l * alpha + wave_sum(ps);
    m_run = m_new;
  }
  chunk_rows_sum<LPR>(acc);
  if (r == 0) {
    const float inv = 1.f / l;
    float out[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) out[e] = acc[e] * inv;
    store8(o + (size_t)inst * D + cg * 8, out);
  }
  if (lane == 0) lse[inst] = (m_run + log2f(l)) * kLn2;
}

// Block b = (patch group mb, head h), heads fastest: its four waves take one
// patch each, m = 4 mb + w, and write dk, dv; the block's share of dq_h goes
// to partial[mb][h][:]. A wave issues all of its loads before its first
// store (loads and stores share one completion counter, so a load issued
// after a store would wait for the store too); with C d <= 6,144 (the
// paper's C = 92 at d = 64) that is a single group of chunks. Each lane
// accumulates ds_c k_c over the rows it holds, and the rows of a chunk are
// summed once at the end.
template <int D>
__global__ __launch_bounds__(256) void attn_agg_bwd_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k, const uint16_t* __restrict__ v,
    const float* __restrict__ o, const uint16_t* __restrict__ dout, const float* __restrict__ lse,
    float* __restrict__ dk, float* __restrict__ dv, float* __restrict__ partial, int M, int H, int C, float c2,
    float scale) {
  constexpr int LPR = D / 8, RPC = 64 / LPR, G = kAggChunkGroup;
  __shared__ __attribute__((aligned(16))) float red[4][D];
  debug_poison_lds(red);
  const int h = blockIdx.x % H, mb = blockIdx.x / H;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int r = lane / LPR, cg = lane % LPR;
  float dqa[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) dqa[e] = 0.f;
  const int m = mb * 4 + wave;
  if (m < M) {  // no early return: the block barrier below needs every wave
    float qv[8];
    widen8(load16(q + (size_t)h * D + cg * 8), qv);
    const int n_chunks = (C + RPC - 1) / RPC;
    const size_t inst = (size_t)m * H + h;
    const size_t base = inst * C * D + lane * 8;
    float g[8], ox[8];
    widen8(load16(dout + inst * D + cg * 8), g);
    const float4 o0 = reinterpret_cast<const float4*>(o + inst * D + cg * 8)[0];
    const float4 o1 = reinterpret_cast<const float4*>(o + inst * D + cg * 8)[1];
    ox[0] = o0.x, ox[1] = o0.y, ox[2] = o0.z, ox[3] = o0.w, ox[4] = o1.x, ox[5] = o1.y, ox[6] = o1.z, ox[7] = o1.w;
    // same product order as dp below: with C = 1 (o = v) ds is then exactly 0
    const float Dm = row_sum<LPR>(dot8(g, ox));
    const float l2 = lse[inst] * kLog2e;
    for (int t0 = 0; t0 < n_chunks; t0 += G) {
      uint4 kr[G], vr[G];
      bool ok[G];
#pragma unroll
      for (int u = 0; u < G; ++u) {
        ok[u] = (t0 + u) * RPC + r < C;
        kr[u] = ok[u] ? load16(k + base + (size_t)(t0 + u) * 512) : make_uint4(0u, 0u, 0u, 0u);
      }
#pragma unroll
      for (int u = 0; u < G; ++u)
        vr[u] = ok[u] ? load16(v + base + (size_t)(t0 + u) * 512) : make_uint4(0u, 0u, 0u, 0u);
#pragma unroll
      for (int u = 0; u < G; ++u) {
        float kx[8], vx[8];
        widen8(kr[u], kx);
        widen8(vr[u], vx);
        const float s = row_sum<LPR>(dot8(kx, qv));
        const float dp = row_sum<LPR>(dot8(g, vx));
        // rows past C (zeros) must add nothing, whatever exp2 gives there
        const float p = ok[u] ? exp2f(s * c2 - l2) : 0.f;
        const float ds = ok[u] ? p * (dp - Dm) : 0.f;
        if (ok[u]) {
          const float f = scale * ds;
          float dkx[8], dvx[8];
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            dkx[e] = f * qv[e];
            dvx[e] = p * g[e];
          }
          store8(dk + base + (size_t)(t0 + u) * 512, dkx);
          store8(dv + base + (size_t)(t0 + u) * 512, dvx);
        }
#pragma unroll
        for (int e = 0; e < 8; ++e) dqa[e] = fmaf(ds, kx[e], dqa[e]);
      }
    }
  }
  chunk_rows_sum<LPR>(dqa);
  if (r == 0) {
#pragma unroll
    for (int e = 0; e < 8; ++e) red[wave][cg * 8 + e] = dqa[e];
  }
  __syncthreads();
  if (threadIdx.x < D) {
    const float s = ((red[0][threadIdx.x] + red[1][threadIdx.x]) + red[2][threadIdx.x]) + red[3][threadIdx.x];
    partial[((size_t)mb * H + h) * D + threadIdx.x] = s;
  }
}

// dq[t] = scale * the sum over patch groups of partial[group][t], t = h*D + e.
// A block of 1,024 threads takes 16 columns; its thread (r, col) sums groups
// r, r+64, r+128, ... in that order, then thread (0, col) adds the 64 sums in
// order of r.
__global__ __launch_bounds__(1024) void attn_agg_dq_kernel(const float* __restrict__ partial, float* __restrict__ dq,
                                                           int groups, int HD, float scale) {
  __shared__ float red[64][17];
  debug_poison_lds(red);
  const int col = threadIdx.x & 15, r = threadIdx.x >> 4;
  const int t = blockIdx.x * 16 + col;
  float s = 0.f;
  if (t < HD) {
#pragma unroll 8
    for (int c = r; c < groups; c += 64) s += partial[(size_t)c * HD + t];
  }
  red[r][col] = s;
  __syncthreads();
  if (r == 0 && t < HD) {
    float tot = 0.f;
#pragma unroll
    for (int i = 0; i < 64; ++i) tot += red[i][col];
    dq[t] = scale * tot;
  }
}

#define VITATTN_AGG_INSTANTIATE(D)                                                                             \
  template __global__ void attn_agg_fwd_kernel<D>(const uint16_t* __restrict__, const uint16_t* __restrict__, \
                                                  const uint16_t* __restrict__, float* __restrict__,          \
                                                  float* __restrict__, int, int, int, float);                 \
  template __global__ void attn_agg_bwd_kernel<D>(                                                             \
      const uint16_t* __restrict__, const uint16_t* __restrict__, const uint16_t* __restrict__,               \
      const float* __restrict__, const uint16_t* __restrict__, const float* __restrict__, float* __restrict__, \
      float* __restrict__, float* __restrict__, int, int, int, float, float);
VITATTN_AGG_INSTANTIATE(64)
VITATTN_AGG_INSTANTIATE(128)
#undef VITATTN_AGG_INSTANTIATE

// dq partials of the backward pass: one per block of four patches
int agg_partials(int M) { return (M + 3) / 4; }

template <int D>
static hipError_t agg_fwd_d(const AggArgs& a) {
  const int MH = a.M * a.H;
  hipLaunchKernelGGL(attn_agg_fwd_kernel<D>, dim3((unsigned)((MH + 3) / 4)), dim3(256), 0, a.stream, a.q, a.k, a.v,
                     a.o_out, a.lse_out, MH, a.H, a.C, a.scale * kLog2e);
  return hipGetLastError();
}

template <int D>
static hipError_t agg_bwd_d(const AggArgs& a) {
  const int parts = agg_partials(a.M);
  hipLaunchKernelGGL(attn_agg_bwd_kernel<D>, dim3((unsigned)(parts * a.H)), dim3(256), 0, a.stream, a.q, a.k, a.v,
                     a.o, a.dout, a.lse, a.dk, a.dv, a.partial, a.M, a.H, a.C, a.scale * kLog2e, a.scale);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int HD = a.H * D;
  hipLaunchKernelGGL(attn_agg_dq_kernel, dim3((unsigned)((HD + 15) / 16)), dim3(1024), 0, a.stream, a.partial, a.dq,
                     parts, HD, a.scale);
  return hipGetLastError();
}

hipError_t launch_agg_fwd(const AggArgs& a) { return a.d == 128 ? agg_fwd_d<128>(a) : agg_fwd_d<64>(a); }
hipError_t launch_agg_bwd(const AggArgs& a) { return a.d == 128 ? agg_bwd_d<128>(a) : agg_bwd_d<64>(a); }

}  // namespace vitattn
