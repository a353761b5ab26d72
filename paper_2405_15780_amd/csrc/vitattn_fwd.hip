// Forward pass of exact non-causal attention for gfx950: tiled online softmax
// (FlashAttention-2, cited by the paper in Sec. II-F) on bf16 matrix cores.
//
// One workgroup = 4 waves = 128 query rows of one (b, h); each wave owns 32
// query rows. The workgroup streams K and V in tiles of 64 keys through a
// double-buffered LDS ring; the next tile is fetched into registers with
// 16-byte coalesced loads while the current one is being used.
//
// Per tile and wave:
//   S^T (keys x queries) = K Q^T   -> each lane holds one query's scores
//   running max / sum per query    -> in-lane, plus one exchange with lane^32
//   P^T = exp2(S^T * scale*log2e - m)
//   O^T (d x queries) += V^T P^T   -> P^T is reused in place as the operand
// The rescale of O by exp2(m_old - m_new) is skipped when no query of the
// wave raised its running max (multiplying by 1 would change nothing), so
// the maximum is always subtracted exactly and the largest P is exactly 1.
#include "vitattn_common.h"
#include "vitattn_launch.h"

namespace vitattn {

constexpr int kFwdWaves = 4;
constexpr int kFwdThreads = 64 * kFwdWaves;
constexpr int kFwdBM = 32 * kFwdWaves;  // query rows per workgroup
constexpr int kFwdBN = 64;              // keys per tile

template <int D>
__global__ __launch_bounds__(kFwdThreads, 2) void attn_fwd_kernel(const uint16_t* __restrict__ q,
                                                                   const uint16_t* __restrict__ k,
                                                                   const uint16_t* __restrict__ v,
                                                                   float* __restrict__ o, float* __restrict__ lse,
                                                                   int N, int n_qtiles, int total, float c) {
  constexpr int TILE_BYTES = kFwdBN * D * 2;
  __shared__ __attribute__((aligned(16))) char smem[2][2][TILE_BYTES];  // [buffer][K, V]

  const int work = xcd_remap(blockIdx.x, total);
  const int bh = work / n_qtiles;
  const int qt = work - bh * n_qtiles;
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6, h = lane >> 5;

  const size_t head_off = (size_t)bh * N * D;
  const uint16_t* Q = q + head_off;
  const uint16_t* K = k + head_off;
  const uint16_t* V = v + head_off;

  // Q fragments of this wave's 32 query rows (B operand of K Q^T).
  const int qrow = qt * kFwdBM + wave * 32 + (lane & 31);
  bf16x8 qf[D / 16];
#pragma unroll
  for (int kk = 0; kk < D / 16; ++kk) {
    uint4 u = make_uint4(0, 0, 0, 0);
    if (qrow < N) u = *reinterpret_cast<const uint4*>(Q + (size_t)qrow * D + 16 * kk + 8 * h);
    qf[kk] = as_bf16x8(u);
  }

  RowFrag<D> kfrag;
  kfrag.init(lane);
  TrFrag<D> vfrag;
  vfrag.init(lane);

  f32x16 oacc[D / 32];
#pragma unroll
  for (int cb = 0; cb < D / 32; ++cb) oacc[cb] = zero16();
  float m_run = -INFINITY;  // running max of scaled logits, log2 units
  float l_part = 0.f;       // this lane's share of the row sum

  const int n_ktiles = (N + kFwdBN - 1) / kFwdBN;
  TileLoader<D, kFwdBN, kFwdThreads> kl, vl;
  kl.load(K, 0, N, tid);
  vl.load(V, 0, N, tid);
  kl.store(smem[0][0], tid);
  vl.store(smem[0][1], tid);
  __syncthreads();

  for (int t = 0; t < n_ktiles; ++t) {
    const int buf = t & 1;
    const bool more = t + 1 < n_ktiles;
    if (more) {
      kl.load(K, (t + 1) * kFwdBN, N, tid);
      vl.load(V, (t + 1) * kFwdBN, N, tid);
    }
    const char* ks = smem[buf][0];
    const char* vs = smem[buf][1];

    // S^T = K Q^T for two blocks of 32 keys
    f32x16 s[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      s[kb] = zero16();
#pragma unroll
      for (int kk = 0; kk < D / 16; ++kk)
        s[kb] = mfma32(lds_frag_row(ks, kb * 32 * 2 * D + kfrag.off[kk]), qf[kk], s[kb]);
    }
    // keys past the end of the sequence (last tile only)
    const int key0 = t * kFwdBN;
    if (key0 + kFwdBN > N) {
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          if (key0 + kb * 32 + acc_row(r, h) >= N) s[kb][r] = -INFINITY;
    }
    // running max per query (lanes l and l^32 share a query)
    float mx = s[0][0];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[kb][r]);
    mx = fmaxf(mx, xor32(mx));
    const float m_tile = mx * c;
    if (__any(m_tile > m_run)) {
      const float m_new = fmaxf(m_run, m_tile);
      const float alpha = __builtin_amdgcn_exp2f(m_run - m_new);
      m_run = m_new;
      l_part *= alpha;
#pragma unroll
      for (int cb = 0; cb < D / 32; ++cb)
#pragma unroll
        for (int r = 0; r < 16; ++r) oacc[cb][r] *= alpha;
    }
    // P^T = exp2(S^T c - m), row sums
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float p = __builtin_amdgcn_exp2f(__builtin_fmaf(s[kb][r], c, -m_run));
        s[kb][r] = p;
        l_part += p;
      }
    // O^T += V^T P^T over 4 contraction steps of 16 keys
#pragma unroll
    for (int kstep = 0; kstep < 4; ++kstep) {
      const bf16x8 pf = acc_to_operand(s[kstep >> 1], kstep & 1);
#pragma unroll
      for (int cb = 0; cb < D / 32; ++cb) oacc[cb] = mfma32(vfrag.load(vs, kstep * 16, cb), pf, oacc[cb]);
    }
    if (more) {
      kl.store(smem[buf ^ 1][0], tid);
      vl.store(smem[buf ^ 1][1], tid);
    }
    __syncthreads();
  }

  // epilogue: O = O^T / l (stored transposed back to [query][d]), LSE in nats.
  // Lanes l and l^32 hold the same query, so both take the same branch.
  const float l = l_part + xor32(l_part);
  if (qrow < N) {
    const float inv = 1.0f / l;
    float* orow = o + head_off + (size_t)qrow * D;
#pragma unroll
    for (int cb = 0; cb < D / 32; ++cb)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        float4 val = make_float4(oacc[cb][4 * g] * inv, oacc[cb][4 * g + 1] * inv, oacc[cb][4 * g + 2] * inv,
                                 oacc[cb][4 * g + 3] * inv);
        *reinterpret_cast<float4*>(orow + 32 * cb + 8 * g + 4 * h) = val;
      }
    if (h == 0) lse[(size_t)bh * N + qrow] = (m_run + __log2f(l)) * kLn2;
  }
}

template <int D>
static hipError_t launch_fwd_d(const FwdArgs& a) {
  const int n_qtiles = (a.N + kFwdBM - 1) / kFwdBM;
  const int total = a.BH * n_qtiles;
  const float c = a.scale * kLog2e;
  hipLaunchKernelGGL(attn_fwd_kernel<D>, dim3(total), dim3(kFwdThreads), 0, a.stream, a.q, a.k, a.v, a.o, a.lse,
                     a.N, n_qtiles, total, c);
  return hipGetLastError();
}

hipError_t launch_fwd(const FwdArgs& a) {
  return a.d == 128 ? launch_fwd_d<128>(a) : launch_fwd_d<64>(a);
}

}  // namespace vitattn
