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
// Many tiny attentions, bound by HBM bandwidth: one wave per (m, h). Scores
// and their dot products are lane-per-key (a lane reads its whole key row);
// the weighted sums over keys are lane-per-column (each V, K, dK, dV row is
// one coalesced 64-lane access) with the key's probability broadcast by
// readlane. Those sums take keys in groups of G, loading the group's rows
// before using any, so that a wave has G row loads in flight rather than one.
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

// dot product of a full d-element bf16 row (this lane's key) with the fp32
// vector x in LDS (the same address for every lane: a broadcast read)
template <int D>
__device__ __forceinline__ float row_dot(const uint16_t* row, const float* x) {
  const uint4* r = reinterpret_cast<const uint4*>(row);
  const float4* xv = reinterpret_cast<const float4*>(x);
  float acc = 0.f;
#pragma unroll
  for (int t = 0; t < D / 8; ++t) {
    const uint4 w = r[t];
    const float4 a = xv[2 * t], b = xv[2 * t + 1];
    acc = fmaf(bf16_lo(w.x), a.x, acc);
    acc = fmaf(bf16_hi(w.x), a.y, acc);
    acc = fmaf(bf16_lo(w.y), a.z, acc);
    acc = fmaf(bf16_hi(w.y), a.w, acc);
    acc = fmaf(bf16_lo(w.z), b.x, acc);
    acc = fmaf(bf16_hi(w.z), b.y, acc);
    acc = fmaf(bf16_lo(w.w), b.z, acc);
    acc = fmaf(bf16_hi(w.w), b.w, acc);
  }
  return acc;
}

// a full d-element bf16 row into registers (8 elements per 16-byte piece)
template <int D>
__device__ __forceinline__ void row_load(const uint16_t* row, uint4 (&r)[D / 8]) {
  const uint4* p = reinterpret_cast<const uint4*>(row);
#pragma unroll
  for (int t = 0; t < D / 8; ++t) r[t] = p[t];
}

// dot product of a row held in registers with the fp32 vector x in LDS
template <int D>
__device__ __forceinline__ float regs_dot(const uint4 (&r)[D / 8], const float* x) {
  const float4* xv = reinterpret_cast<const float4*>(x);
  float acc = 0.f;
#pragma unroll
  for (int t = 0; t < D / 8; ++t) {
    const uint4 w = r[t];
    const float4 a = xv[2 * t], b = xv[2 * t + 1];
    acc = fmaf(bf16_lo(w.x), a.x, acc);
    acc = fmaf(bf16_hi(w.x), a.y, acc);
    acc = fmaf(bf16_lo(w.y), a.z, acc);
    acc = fmaf(bf16_hi(w.y), a.w, acc);
    acc = fmaf(bf16_lo(w.z), b.x, acc);
    acc = fmaf(bf16_hi(w.z), b.y, acc);
    acc = fmaf(bf16_lo(w.w), b.z, acc);
    acc = fmaf(bf16_hi(w.w), b.w, acc);
  }
  return acc;
}

// acc[e] += f * row[e] for a bf16 row held in registers
template <int D>
__device__ __forceinline__ void regs_axpy(float f, const uint4 (&r)[D / 8], float (&acc)[D]) {
#pragma unroll
  for (int t = 0; t < D / 8; ++t) {
    const uint4 w = r[t];
    acc[8 * t + 0] = fmaf(f, bf16_lo(w.x), acc[8 * t + 0]);
    acc[8 * t + 1] = fmaf(f, bf16_hi(w.x), acc[8 * t + 1]);
    acc[8 * t + 2] = fmaf(f, bf16_lo(w.y), acc[8 * t + 2]);
    acc[8 * t + 3] = fmaf(f, bf16_hi(w.y), acc[8 * t + 3]);
    acc[8 * t + 4] = fmaf(f, bf16_lo(w.z), acc[8 * t + 4]);
    acc[8 * t + 5] = fmaf(f, bf16_hi(w.z), acc[8 * t + 5]);
    acc[8 * t + 6] = fmaf(f, bf16_lo(w.w), acc[8 * t + 6]);
    acc[8 * t + 7] = fmaf(f, bf16_hi(w.w), acc[8 * t + 7]);
  }
}

// Sum of a 64-column per-lane vector over the wave's 64 lanes, by recursive
// halving: at each of six steps a lane keeps half of its columns, receives
// the partner's (lane ^ o) share of that half and adds; lane l ends with
// column l's sum (its kept half is the upper one exactly when bit o of l is
// set, so the surviving column index spells out l). 63 exchanges in all.
__device__ __forceinline__ float wave_column_sums(float (&acc)[64], int lane) {
  static_for<0, 6>([&](auto SC) __attribute__((always_inline)) {
    constexpr int o = 32 >> decltype(SC)::value, half = o;  // columns left: 2*half -> half
    const bool upper = (lane & o) != 0;
#pragma unroll
    for (int i = 0; i < half; ++i) {
      const float send = upper ? acc[i] : acc[i + half];
      const float keep = upper ? acc[i + half] : acc[i];
      acc[i] = keep + __shfl_xor(send, o);
    }
  });
  return acc[0];
}

// this lane's E = D/64 consecutive columns of a bf16 row, widened
template <int D>
__device__ __forceinline__ void row_cols(const uint16_t* row, int lane, float (&out)[D / 64]) {
  if constexpr (D == 128) {
    const uint32_t w = reinterpret_cast<const uint32_t*>(row)[lane];
    out[0] = bf16_lo(w);
    out[1] = bf16_hi(w);
  } else {
    out[0] = __uint_as_float((uint32_t)row[lane] << 16);
  }
}

// a bf16 d-vector widened into this wave's LDS slot (each lane its columns)
template <int D>
__device__ __forceinline__ void stage_vec(const uint16_t* src, float* dst, int lane) {
  float x[D / 64];
  row_cols<D>(src, lane, x);
#pragma unroll
  for (int e = 0; e < D / 64; ++e) dst[lane * (D / 64) + e] = x[e];
}

}  // namespace

template <int D>
__global__ __launch_bounds__(256) void attn_agg_fwd_kernel(const uint16_t* __restrict__ q,
                                                           const uint16_t* __restrict__ k,
                                                           const uint16_t* __restrict__ v, float* __restrict__ o,
                                                           float* __restrict__ lse, int MH, int H, int C, float c2) {
  constexpr int E = D / 64;  // columns per lane
  __shared__ __attribute__((aligned(16))) float qs[4][D];
  const int wave = threadIdx.x >> 6;
  const int inst = blockIdx.x * 4 + wave;
  if (inst >= MH) return;  // whole waves exit together; no block barrier follows
  const int lane = threadIdx.x & 63;
  const int h = inst % H;
  float* qx = qs[wave];
  stage_vec<D>(q + (size_t)h * D, qx, lane);  // a wave's own LDS writes precede its reads
  const uint16_t* kb = k + (size_t)inst * C * D;
  const uint16_t* vb = v + (size_t)inst * C * D;

  float m_run = -INFINITY, l = 0.f;  // log2 units
  float acc[E];
#pragma unroll
  for (int e = 0; e < E; ++e) acc[e] = 0.f;
  for (int c0 = 0; c0 < C; c0 += 64) {
    const int c = c0 + lane;
    const float s = c < C ? row_dot<D>(kb + (size_t)c * D, qx) * c2 : -INFINITY;
    const float m_new = fmaxf(m_run, wave_max(s));
    const float alpha = exp2f(m_run - m_new);
    const float p = c < C ? exp2f(s - m_new) : 0.f;
    l = l * alpha + wave_sum(p);
#pragma unroll
    for (int e = 0; e < E; ++e) acc[e] *= alpha;
    const int n = min(64, C - c0);
    const auto key = [&](int j, const float (&vc)[E]) {
      const float pj = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, p), j));
#pragma unroll
      for (int e = 0; e < E; ++e) acc[e] = fmaf(pj, vc[e], acc[e]);
    };
    int j = 0;
    for (; j + kAggGroup <= n; j += kAggGroup) {
      float vc[kAggGroup][E];
#pragma unroll
      for (int u = 0; u < kAggGroup; ++u) row_cols<D>(vb + (size_t)(c0 + j + u) * D, lane, vc[u]);
#pragma unroll
      for (int u = 0; u < kAggGroup; ++u) key(j + u, vc[u]);
    }
    for (; j < n; ++j) {
      float vc[E];
      row_cols<D>(vb + (size_t)(c0 + j) * D, lane, vc);
      key(j, vc);
    }
    m_run = m_new;
  }
  const float inv = 1.f / l;
#pragma unroll
  for (int e = 0; e < E; ++e) o[(size_t)inst * D + lane * E + e] = acc[e] * inv;
  if (lane == 0) lse[inst] = (m_run + log2f(l)) * kLn2;
}

// Block (chunk, h): waves take patches m = chunk*per + w, + 4, ... below
// (chunk+1)*per and write dk, dv; the block's share of dq_h goes to
// partial[chunk][h][:]. For d = 64 a lane accumulates ds_c k_c of its own
// keys from the K row it already holds for the score (K is read once), and
// the wave's columns are summed at the end; wider heads sum dq column-wise
// from a second, coalesced read of each K row.
template <int D>
__global__ __launch_bounds__(256) void attn_agg_bwd_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k, const uint16_t* __restrict__ v,
    const float* __restrict__ o, const uint16_t* __restrict__ dout, const float* __restrict__ lse,
    float* __restrict__ dk, float* __restrict__ dv, float* __restrict__ partial, int M, int H, int C, int per,
    float c2, float scale) {
  constexpr int E = D / 64;
  __shared__ __attribute__((aligned(16))) float red[4][D];
  __shared__ __attribute__((aligned(16))) float qs[D];
  __shared__ __attribute__((aligned(16))) float gs[4][D];
  const int chunk = blockIdx.x, h = blockIdx.y;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  if (wave == 0) stage_vec<D>(q + (size_t)h * D, qs, lane);
  __syncthreads();
  const float* qx = qs;
  float* gx = gs[wave];
  constexpr bool LANE_DQ = D == 64;
  float dq[E];
#pragma unroll
  for (int e = 0; e < E; ++e) dq[e] = 0.f;
  float dql[LANE_DQ ? D : 1];  // LANE_DQ: this lane's keys' share of dq, all columns
#pragma unroll
  for (int e = 0; e < (LANE_DQ ? D : 1); ++e) dql[e] = 0.f;
  const int m_end = min(M, (chunk + 1) * per);
  for (int m = chunk * per + wave; m < m_end; m += 4) {
    const size_t inst = (size_t)m * H + h;
    const uint16_t* kb = k + inst * C * D;
    const uint16_t* vb = v + inst * C * D;
    float* dkb = dk + inst * C * D;
    float* dvb = dv + inst * C * D;
    // dO of this instance: in the wave's LDS slot (for dp) and its own columns
    stage_vec<D>(dout + inst * D, gx, lane);
    float g[E], oc[E];
    row_cols<D>(dout + inst * D, lane, g);
#pragma unroll
    for (int e = 0; e < E; ++e) oc[e] = o[inst * D + lane * E + e];
    float dpart = 0.f;
#pragma unroll
    for (int e = 0; e < E; ++e) dpart = fmaf(g[e], oc[e], dpart);
    const float Dm = wave_sum(dpart);
    const float l2 = lse[inst] * kLog2e;
    for (int c0 = 0; c0 < C; c0 += 64) {
      const int c = c0 + lane;
      float p = 0.f, ds = 0.f;
      if (c < C) {
        if constexpr (LANE_DQ) {
          // dP first, so that only one of the two rows is live at a time
          const float dp = row_dot<D>(vb + (size_t)c * D, gx);
          uint4 kr[D / 8];
          row_load<D>(kb + (size_t)c * D, kr);
          p = exp2f(regs_dot<D>(kr, qx) * c2 - l2);
          ds = p * (dp - Dm);
          regs_axpy<D>(ds, kr, dql);
        } else {
          p = exp2f(row_dot<D>(kb + (size_t)c * D, qx) * c2 - l2);
          ds = p * (row_dot<D>(vb + (size_t)c * D, gx) - Dm);
        }
      }
      const int n = min(64, C - c0);
      const auto key = [&](int j, const float (&kc)[E]) {
        const float pj = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, p), j));
        const float dsj = __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, ds), j));
        const size_t row = (size_t)(c0 + j) * D;
#pragma unroll
        for (int e = 0; e < E; ++e) {
          dkb[row + lane * E + e] = scale * dsj * qx[lane * E + e];
          dvb[row + lane * E + e] = pj * g[e];
          if constexpr (!LANE_DQ) dq[e] = fmaf(dsj, kc[e], dq[e]);
        }
      };
      if constexpr (LANE_DQ) {  // stores only: dq came from the registers above
        const float none[E] = {};
        for (int j = 0; j < n; ++j) key(j, none);
        continue;
      }
      int j = 0;
      for (; j + kAggGroup <= n; j += kAggGroup) {
        float kc[kAggGroup][E];
#pragma unroll
        for (int u = 0; u < kAggGroup; ++u) row_cols<D>(kb + (size_t)(c0 + j + u) * D, lane, kc[u]);
#pragma unroll
        for (int u = 0; u < kAggGroup; ++u) key(j + u, kc[u]);
      }
      for (; j < n; ++j) {
        float kc[E];
        row_cols<D>(kb + (size_t)(c0 + j) * D, lane, kc);
        key(j, kc);
      }
    }
  }
  if constexpr (LANE_DQ) dq[0] = wave_column_sums(dql, lane);  // E = 1: lane l holds column l
#pragma unroll
  for (int e = 0; e < E; ++e) red[wave][lane * E + e] = dq[e];
  __syncthreads();
  if (threadIdx.x < D) {
    const float s = ((red[0][threadIdx.x] + red[1][threadIdx.x]) + red[2][threadIdx.x]) + red[3][threadIdx.x];
    partial[((size_t)chunk * H + h) * D + threadIdx.x] = s;
  }
}

// dq[t] = scale * the sum over chunks of partial[chunk][t], t = h*D + e. A
// block takes 16 columns; its thread (r, col) sums chunks r, r+16, r+32, ...
// in that order, then thread (0, col) adds the 16 sums in order of r.
__global__ __launch_bounds__(256) void attn_agg_dq_kernel(const float* __restrict__ partial, float* __restrict__ dq,
                                                          int chunks, int HD, float scale) {
  __shared__ float red[16][17];
  const int col = threadIdx.x & 15, r = threadIdx.x >> 4;
  const int t = blockIdx.x * 16 + col;
  float s = 0.f;
  if (t < HD) {
#pragma unroll 8
    for (int c = r; c < chunks; c += 16) s += partial[(size_t)c * HD + t];
  }
  red[r][col] = s;
  __syncthreads();
  if (r == 0 && t < HD) {
    float tot = 0.f;
#pragma unroll
    for (int i = 0; i < 16; ++i) tot += red[i][col];
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
      float* __restrict__, float* __restrict__, int, int, int, int, float, float);
VITATTN_AGG_INSTANTIATE(64)
VITATTN_AGG_INSTANTIATE(128)
#undef VITATTN_AGG_INSTANTIATE

// blocks along M in the backward pass: about kAggTargetBlocks blocks in all
int agg_chunks(int M, int H) {
  const int target = kAggTargetBlocks / H > 1 ? kAggTargetBlocks / H : 1;
  const int c = target < kAggMaxChunks ? target : kAggMaxChunks;
  return M < c ? M : c;
}

template <int D>
static hipError_t agg_fwd_d(const AggArgs& a) {
  const int MH = a.M * a.H;
  hipLaunchKernelGGL(attn_agg_fwd_kernel<D>, dim3((unsigned)((MH + 3) / 4)), dim3(256), 0, a.stream, a.q, a.k, a.v,
                     a.o_out, a.lse_out, MH, a.H, a.C, a.scale * kLog2e);
  return hipGetLastError();
}

template <int D>
static hipError_t agg_bwd_d(const AggArgs& a) {
  const int chunks = agg_chunks(a.M, a.H);
  const int per = (a.M + chunks - 1) / chunks;
  hipLaunchKernelGGL(attn_agg_bwd_kernel<D>, dim3((unsigned)chunks, (unsigned)a.H), dim3(256), 0, a.stream, a.q, a.k,
                     a.v, a.o, a.dout, a.lse, a.dk, a.dv, a.partial, a.M, a.H, a.C, per, a.scale * kLog2e, a.scale);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int HD = a.H * D;
  hipLaunchKernelGGL(attn_agg_dq_kernel, dim3((unsigned)((HD + 15) / 16)), dim3(256), 0, a.stream, a.partial, a.dq,
                     chunks, HD, a.scale);
  return hipGetLastError();
}

hipError_t launch_agg_fwd(const AggArgs& a) { return a.d == 128 ? agg_fwd_d<128>(a) : agg_fwd_d<64>(a); }
hipError_t launch_agg_bwd(const AggArgs& a) { return a.d == 128 ? agg_bwd_d<128>(a) : agg_bwd_d<64>(a); }

}  // namespace vitattn
