// Backward pass of exact non-causal attention for gfx950 (FlashAttention-2's
// backward, cited by the paper in Sec. II-F): P is recomputed from Q, K and
// the saved logsumexp, never stored.
//
//   1. preprocess:  D_i = sum_c dO_ic O_ic                (HBM-bound)
//   2. dK/dV kernel: one workgroup per 128 keys (32 per wave, K and V held in
//      registers); streams Q, dO, LSE and D in tiles of 64 queries:
//        S = Q K^T, P = exp2(S*scale*log2e - LSE*log2e)
//        dV^T += dO^T P,  dP = dO V^T,  dS = P o (dP - D),  dK^T += Q^T dS
//   3. dQ kernel: one workgroup per 128 queries (32 per wave, Q and dO held in
//      registers); streams K and V in tiles of 64 keys:
//        S^T = K Q^T, P^T, dP^T = V dO^T, dS^T, dQ^T += K^T dS^T
// Splitting dQ from dK/dV costs one extra recomputation of S and dP but needs
// no atomics, so results are deterministic.
#include "vitattn_common.h"
#include "vitattn_launch.h"

namespace vitattn {

constexpr int kBwdWaves = 4;
constexpr int kBwdThreads = 64 * kBwdWaves;

// ------------------------------------------------------------------ preprocess

template <int D>
__global__ __launch_bounds__(256) void attn_bwd_rowdot_kernel(const uint16_t* __restrict__ dout,
                                                              const float* __restrict__ o, float* __restrict__ drow,
                                                              long rows) {
  constexpr int LPR = D / 8;  // lanes per row, 8 elements each
  const long row = (long)blockIdx.x * (256 / LPR) + threadIdx.x / LPR;
  const int part = threadIdx.x % LPR;
  float acc = 0.f;
  if (row < rows) {
    const uint4 g = *reinterpret_cast<const uint4*>(dout + row * D + part * 8);
    const float4 o0 = *reinterpret_cast<const float4*>(o + row * D + part * 8);
    const float4 o1 = *reinterpret_cast<const float4*>(o + row * D + part * 8 + 4);
    const bf16x8 gb = as_bf16x8(g);
    acc = (float)gb[0] * o0.x + (float)gb[1] * o0.y + (float)gb[2] * o0.z + (float)gb[3] * o0.w +
          (float)gb[4] * o1.x + (float)gb[5] * o1.y + (float)gb[6] * o1.z + (float)gb[7] * o1.w;
  }
#pragma unroll
  for (int m = LPR / 2; m >= 1; m >>= 1) acc += __shfl_xor(acc, m, 64);
  if (row < rows && part == 0) drow[row] = acc;
}

// ------------------------------------------------------------------ dK / dV

constexpr int kDkvBK = 32 * kBwdWaves;  // keys per workgroup
constexpr int kDkvBQ = 64;              // queries per streamed tile

// Per-row statistics of a query tile (LSE in log2 units, and D), staged
// through registers like the bf16 tiles. Rows at or past N get LSE = +inf
// (so P = 0) and D = 0.
struct RowStatLoader {
  float val;
  __device__ __forceinline__ void load(const float* __restrict__ lse, const float* __restrict__ drow, int row0,
                                       int N, int tid) {
    if (tid < kDkvBQ) {
      const int row = row0 + tid;
      val = row < N ? lse[row] * kLog2e : INFINITY;
    } else if (tid < 2 * kDkvBQ) {
      const int row = row0 + tid - kDkvBQ;
      val = row < N ? drow[row] : 0.f;
    }
  }
  __device__ __forceinline__ void store(float* s, int tid) const {
    if (tid < 2 * kDkvBQ) s[tid] = val;
  }
};

template <int D>
__global__ __launch_bounds__(kBwdThreads, 1) void attn_bwd_dkdv_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k, const uint16_t* __restrict__ v,
    const uint16_t* __restrict__ dout, const float* __restrict__ lse, const float* __restrict__ drow,
    float* __restrict__ dk, float* __restrict__ dv, int N, int n_ktiles, int total, float c, float scale) {
  constexpr int TILE_BYTES = kDkvBQ * D * 2;
  __shared__ __attribute__((aligned(16))) char smem[2][2][TILE_BYTES];  // [buffer][Q, dO]
  __shared__ __attribute__((aligned(16))) float sstat[2][2 * kDkvBQ];    // [buffer][LSE2 | D]

  const int work = xcd_remap(blockIdx.x, total);
  const int bh = work / n_ktiles;
  const int kt = work - bh * n_ktiles;
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6, h = lane >> 5;

  const size_t head_off = (size_t)bh * N * D;
  const uint16_t* Q = q + head_off;
  const uint16_t* dO = dout + head_off;
  const float* L = lse + (size_t)bh * N;
  const float* Dr = drow + (size_t)bh * N;

  // this wave's 32 keys: K and V fragments as B operands (columns = keys)
  const int key = kt * kDkvBK + wave * 32 + (lane & 31);
  bf16x8 kf[D / 16], vf[D / 16];
#pragma unroll
  for (int kk = 0; kk < D / 16; ++kk) {
    uint4 a = make_uint4(0, 0, 0, 0), b = make_uint4(0, 0, 0, 0);
    if (key < N) {
      a = *reinterpret_cast<const uint4*>(k + head_off + (size_t)key * D + 16 * kk + 8 * h);
      b = *reinterpret_cast<const uint4*>(v + head_off + (size_t)key * D + 16 * kk + 8 * h);
    }
    kf[kk] = as_bf16x8(a);
    vf[kk] = as_bf16x8(b);
  }

  RowFrag<D> rf;
  rf.init(lane);
  TrFrag<D> tf;
  tf.init(lane);

  f32x16 dkacc[D / 32], dvacc[D / 32];
#pragma unroll
  for (int cb = 0; cb < D / 32; ++cb) {
    dkacc[cb] = zero16();
    dvacc[cb] = zero16();
  }

  const int n_qt = (N + kDkvBQ - 1) / kDkvBQ;
  TileLoader<D, kDkvBQ, kBwdThreads> ql, gl;
  RowStatLoader sl;
  ql.load(Q, 0, N, tid);
  gl.load(dO, 0, N, tid);
  sl.load(L, Dr, 0, N, tid);
  ql.store(smem[0][0], tid);
  gl.store(smem[0][1], tid);
  sl.store(sstat[0], tid);
  __syncthreads();

  for (int t = 0; t < n_qt; ++t) {
    const int buf = t & 1;
    const bool more = t + 1 < n_qt;
    if (more) {
      ql.load(Q, (t + 1) * kDkvBQ, N, tid);
      gl.load(dO, (t + 1) * kDkvBQ, N, tid);
      sl.load(L, Dr, (t + 1) * kDkvBQ, N, tid);
    }
    const char* qs = smem[buf][0];
    const char* gs = smem[buf][1];
    const float* st = sstat[buf];

#pragma unroll
    for (int qb = 0; qb < kDkvBQ / 32; ++qb) {
      // S = Q K^T (rows = queries, columns = this wave's keys)
      f32x16 s = zero16();
#pragma unroll
      for (int kk = 0; kk < D / 16; ++kk) s = mfma32(lds_frag_row(qs, qb * 32 * 2 * D + rf.off[kk]), kf[kk], s);
      // P = exp2(S c - LSE2[row])
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const float4 l4 = *reinterpret_cast<const float4*>(st + qb * 32 + 8 * g + 4 * h);
        s[4 * g + 0] = __builtin_amdgcn_exp2f(__builtin_fmaf(s[4 * g + 0], c, -l4.x));
        s[4 * g + 1] = __builtin_amdgcn_exp2f(__builtin_fmaf(s[4 * g + 1], c, -l4.y));
        s[4 * g + 2] = __builtin_amdgcn_exp2f(__builtin_fmaf(s[4 * g + 2], c, -l4.z));
        s[4 * g + 3] = __builtin_amdgcn_exp2f(__builtin_fmaf(s[4 * g + 3], c, -l4.w));
      }
      // dV^T += dO^T P
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
        const bf16x8 pf = acc_to_operand(s, ks);
#pragma unroll
        for (int cb = 0; cb < D / 32; ++cb) dvacc[cb] = mfma32(tf.load(gs, qb * 32 + 16 * ks, cb), pf, dvacc[cb]);
      }
      // dP = dO V^T
      f32x16 dp = zero16();
#pragma unroll
      for (int kk = 0; kk < D / 16; ++kk) dp = mfma32(lds_frag_row(gs, qb * 32 * 2 * D + rf.off[kk]), vf[kk], dp);
      // dS = P o (dP - D[row])
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const float4 d4 = *reinterpret_cast<const float4*>(st + kDkvBQ + qb * 32 + 8 * g + 4 * h);
        dp[4 * g + 0] = s[4 * g + 0] * (dp[4 * g + 0] - d4.x);
        dp[4 * g + 1] = s[4 * g + 1] * (dp[4 * g + 1] - d4.y);
        dp[4 * g + 2] = s[4 * g + 2] * (dp[4 * g + 2] - d4.z);
        dp[4 * g + 3] = s[4 * g + 3] * (dp[4 * g + 3] - d4.w);
      }
      // dK^T += Q^T dS
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
        const bf16x8 df = acc_to_operand(dp, ks);
#pragma unroll
        for (int cb = 0; cb < D / 32; ++cb) dkacc[cb] = mfma32(tf.load(qs, qb * 32 + 16 * ks, cb), df, dkacc[cb]);
      }
    }
    if (more) {
      ql.store(smem[buf ^ 1][0], tid);
      gl.store(smem[buf ^ 1][1], tid);
      sl.store(sstat[buf ^ 1], tid);
    }
    __syncthreads();
  }

  if (key < N) {
    float* dkrow = dk + head_off + (size_t)key * D;
    float* dvrow = dv + head_off + (size_t)key * D;
#pragma unroll
    for (int cb = 0; cb < D / 32; ++cb)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int col = 32 * cb + 8 * g + 4 * h;
        *reinterpret_cast<float4*>(dkrow + col) =
            make_float4(dkacc[cb][4 * g] * scale, dkacc[cb][4 * g + 1] * scale, dkacc[cb][4 * g + 2] * scale,
                        dkacc[cb][4 * g + 3] * scale);
        *reinterpret_cast<float4*>(dvrow + col) =
            make_float4(dvacc[cb][4 * g], dvacc[cb][4 * g + 1], dvacc[cb][4 * g + 2], dvacc[cb][4 * g + 3]);
      }
  }
}

// ------------------------------------------------------------------ dQ

constexpr int kDqBM = 32 * kBwdWaves;  // queries per workgroup
constexpr int kDqBN = 64;              // keys per streamed tile

template <int D>
__global__ __launch_bounds__(kBwdThreads, 2) void attn_bwd_dq_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k, const uint16_t* __restrict__ v,
    const uint16_t* __restrict__ dout, const float* __restrict__ lse, const float* __restrict__ drow,
    float* __restrict__ dq, int N, int n_qtiles, int total, float c, float scale) {
  constexpr int TILE_BYTES = kDqBN * D * 2;
  __shared__ __attribute__((aligned(16))) char smem[2][2][TILE_BYTES];  // [buffer][K, V]

  const int work = xcd_remap(blockIdx.x, total);
  const int bh = work / n_qtiles;
  const int qt = work - bh * n_qtiles;
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6, h = lane >> 5;

  const size_t head_off = (size_t)bh * N * D;
  const uint16_t* K = k + head_off;
  const uint16_t* V = v + head_off;

  const int qrow = qt * kDqBM + wave * 32 + (lane & 31);
  bf16x8 qf[D / 16], gf[D / 16];
#pragma unroll
  for (int kk = 0; kk < D / 16; ++kk) {
    uint4 a = make_uint4(0, 0, 0, 0), b = make_uint4(0, 0, 0, 0);
    if (qrow < N) {
      a = *reinterpret_cast<const uint4*>(q + head_off + (size_t)qrow * D + 16 * kk + 8 * h);
      b = *reinterpret_cast<const uint4*>(dout + head_off + (size_t)qrow * D + 16 * kk + 8 * h);
    }
    qf[kk] = as_bf16x8(a);
    gf[kk] = as_bf16x8(b);
  }
  const float lse2 = qrow < N ? lse[(size_t)bh * N + qrow] * kLog2e : INFINITY;
  const float dval = qrow < N ? drow[(size_t)bh * N + qrow] : 0.f;

  RowFrag<D> rf;
  rf.init(lane);
  TrFrag<D> tf;
  tf.init(lane);

  f32x16 dqacc[D / 32];
#pragma unroll
  for (int cb = 0; cb < D / 32; ++cb) dqacc[cb] = zero16();

  const int n_kt = (N + kDqBN - 1) / kDqBN;
  TileLoader<D, kDqBN, kBwdThreads> kl, vl;
  kl.load(K, 0, N, tid);
  vl.load(V, 0, N, tid);
  kl.store(smem[0][0], tid);
  vl.store(smem[0][1], tid);
  __syncthreads();

  for (int t = 0; t < n_kt; ++t) {
    const int buf = t & 1;
    const bool more = t + 1 < n_kt;
    if (more) {
      kl.load(K, (t + 1) * kDqBN, N, tid);
      vl.load(V, (t + 1) * kDqBN, N, tid);
    }
    const char* ks = smem[buf][0];
    const char* vs = smem[buf][1];
    const int key0 = t * kDqBN;
    const bool tail = key0 + kDqBN > N;

#pragma unroll
    for (int kb = 0; kb < kDqBN / 32; ++kb) {
      // S^T = K Q^T, P^T = exp2(S^T c - LSE2)
      f32x16 s = zero16();
#pragma unroll
      for (int kk = 0; kk < D / 16; ++kk) s = mfma32(lds_frag_row(ks, kb * 32 * 2 * D + rf.off[kk]), qf[kk], s);
#pragma unroll
      for (int r = 0; r < 16; ++r) s[r] = __builtin_amdgcn_exp2f(__builtin_fmaf(s[r], c, -lse2));
      if (tail) {
#pragma unroll
        for (int r = 0; r < 16; ++r)
          if (key0 + kb * 32 + acc_row(r, h) >= N) s[r] = 0.f;
      }
      // dP^T = V dO^T, dS^T = P^T o (dP^T - D)
      f32x16 dp = zero16();
#pragma unroll
      for (int kk = 0; kk < D / 16; ++kk) dp = mfma32(lds_frag_row(vs, kb * 32 * 2 * D + rf.off[kk]), gf[kk], dp);
#pragma unroll
      for (int r = 0; r < 16; ++r) dp[r] = s[r] * (dp[r] - dval);
      // dQ^T += K^T dS^T
#pragma unroll
      for (int ks2 = 0; ks2 < 2; ++ks2) {
        const bf16x8 df = acc_to_operand(dp, ks2);
#pragma unroll
        for (int cb = 0; cb < D / 32; ++cb) dqacc[cb] = mfma32(tf.load(ks, kb * 32 + 16 * ks2, cb), df, dqacc[cb]);
      }
    }
    if (more) {
      kl.store(smem[buf ^ 1][0], tid);
      vl.store(smem[buf ^ 1][1], tid);
    }
    __syncthreads();
  }

  if (qrow < N) {
    float* row = dq + head_off + (size_t)qrow * D;
#pragma unroll
    for (int cb = 0; cb < D / 32; ++cb)
#pragma unroll
      for (int g = 0; g < 4; ++g)
        *reinterpret_cast<float4*>(row + 32 * cb + 8 * g + 4 * h) =
            make_float4(dqacc[cb][4 * g] * scale, dqacc[cb][4 * g + 1] * scale, dqacc[cb][4 * g + 2] * scale,
                        dqacc[cb][4 * g + 3] * scale);
  }
}

// ------------------------------------------------------------------ launch

template <int D>
static hipError_t rowdot_d(const BwdArgs& a) {
  const long rows = (long)a.BH * a.N;
  constexpr int rows_per_block = 256 / (D / 8);
  hipLaunchKernelGGL(attn_bwd_rowdot_kernel<D>, dim3((unsigned)((rows + rows_per_block - 1) / rows_per_block)),
                     dim3(256), 0, a.stream, a.dout, a.o, a.drow, rows);
  return hipGetLastError();
}

template <int D>
static hipError_t dkdv_d(const BwdArgs& a) {
  const int n_kt = (a.N + kDkvBK - 1) / kDkvBK;
  const int total = a.BH * n_kt;
  hipLaunchKernelGGL(attn_bwd_dkdv_kernel<D>, dim3(total), dim3(kBwdThreads), 0, a.stream, a.q, a.k, a.v, a.dout,
                     a.lse, a.drow, a.dk, a.dv, a.N, n_kt, total, a.scale * kLog2e, a.scale);
  return hipGetLastError();
}

template <int D>
static hipError_t dq_d(const BwdArgs& a) {
  const int n_qt = (a.N + kDqBM - 1) / kDqBM;
  const int total = a.BH * n_qt;
  hipLaunchKernelGGL(attn_bwd_dq_kernel<D>, dim3(total), dim3(kBwdThreads), 0, a.stream, a.q, a.k, a.v, a.dout,
                     a.lse, a.drow, a.dq, a.N, n_qt, total, a.scale * kLog2e, a.scale);
  return hipGetLastError();
}

hipError_t launch_bwd_rowdot(const BwdArgs& a) { return a.d == 128 ? rowdot_d<128>(a) : rowdot_d<64>(a); }
hipError_t launch_bwd_dkdv(const BwdArgs& a) { return a.d == 128 ? dkdv_d<128>(a) : dkdv_d<64>(a); }
hipError_t launch_bwd_dq(const BwdArgs& a) { return a.d == 128 ? dq_d<128>(a) : dq_d<64>(a); }

hipError_t launch_bwd(const BwdArgs& a) {
  hipError_t e = launch_bwd_rowdot(a);
  if (e == hipSuccess) e = launch_bwd_dkdv(a);
  if (e == hipSuccess) e = launch_bwd_dq(a);
  return e;
}

}  // namespace vitattn
