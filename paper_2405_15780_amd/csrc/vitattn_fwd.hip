// Forward pass of exact non-causal attention for gfx950: tiled online softmax
// (FlashAttention-2, cited by the paper in Sec. II-F) on bf16 matrix cores.
//
// One workgroup = NW waves = 32*NW query rows of one (b, h); each wave owns
// 32 query rows and keeps their Q fragments in registers. K and V stream
// through LDS in tiles of 32*KB keys, copied straight from HBM into the
// swizzled LDS layout by buffer loads (rows past the end arrive as zeros).
//
// Per tile and wave:
//   S^T (keys x queries) = K Q^T   -> each lane holds one query's scores
//   running max / sum per query    -> in-lane, plus one exchange with lane^32
//   P^T = exp2(S^T * scale*log2e - m)
//   O^T (d x queries) += V^T P^T   -> P^T is reused in place as the operand
//
// Operands may have any batch / head / row strides (rows 16-byte aligned): the
// kernel only forms addresses from them. The tile width D is 64, 96, 128 or
// 160; for a head dim d below D the columns past d are loaded as zeros (they
// add nothing to the scores) and never stored. The scores contract over the
// KS 16-column steps of d that hold data (D/16, or 5 for d <= 80 in the
// 96-wide tile): the steps past them would add exact zeros.
//
// Software pipeline across tiles: the scores of tile j+1 are computed on the
// matrix cores while the vector units turn tile j's scores into
// probabilities. K therefore runs one tile ahead of V, in two LDS rings of
// two slots: iteration j reads K_{j+1} and V_j and refills the slots of K_j
// and V_{j-1} with K_{j+2} and V_{j+1}. The tile loop is unrolled by two so
// that every LDS address is a lane offset plus a constant.
//
// Software pipeline within a tile: one stream of score ops then PV ops, each
// op's LDS operand read two ops ahead, with the vector work cut into slices
// placed between the ops and scheduling fences pinning that order. The
// matrix cores only stay busy while each wave's vector work is spread thinly
// and evenly over its own op stream, so the exponentials of tile j cover both
// the score ops of tile j+1 and the PV ops of tile j (each 16-key step's
// probabilities finish two ops before the PV op that reads them), and the
// row max of tile j+1 is taken in the last PV slots.
//
// The row sum adds the fp32 probabilities in two partial sums (plain adds:
// a v_dot2 over the bf16 pairs would compete with the matrix cores). The
// rescale of O by exp2(m_old - m_new) is skipped when no query of the wave
// raised its running max (multiplying by 1 would change nothing). The
// running max m is kept pre-multiplied by the scale (m = fl(max * c)) and
// subtracted inside one FMA, exp2(fma(s, c, -m)), so the largest P is 1 up
// to the rounding of that product (one fp32 ulp of the scaled logit).
#include <atomic>
#include <type_traits>

#include "vitattn_common.h"
#include "vitattn_launch.h"

namespace vitattn {

// Score e (of 16*KB per lane) is exponentiated in slot e*W/(16*KB); the
// probabilities of 16-key step t (scores 8t .. 8t+7) are consumed by the PV
// op at NS + CPB*t and must be complete two slots earlier.
constexpr bool exp_schedule_ok(int NS, int CPB, int KB, int W) {
  const int ne = 16 * KB;
  for (int t = 0; t < 2 * KB; ++t)
    if ((8 * t + 7) * W / ne > NS + CPB * t - 2) return false;
  return true;
}

// Widest exponential window (at most NOPS - 5 slots, which leaves the last
// slots to the row max of the next tile) that keeps exp_schedule_ok.
constexpr int exp_window(int NS, int CPB, int KB, int NOPS) {
  int w = NOPS - 5;
  while (w > 1 && !exp_schedule_ok(NS, CPB, KB, w)) --w;
  return w;
}

template <int D, int KB, int NW, int MINW, int KS = D / 16>
__global__ __launch_bounds__(64 * NW, MINW) void attn_fwd_kernel(const uint16_t* __restrict__ q,
                                                                 const uint16_t* __restrict__ k,
                                                                 const uint16_t* __restrict__ v,
                                                                 float* __restrict__ o, float* __restrict__ lse,
                                                                 const Map mq, const Map mk, const Map mv,
                                                                 const Map mo, int H, int dr, int Nq, int Nk,
                                                                 int n_qtiles, int total, float c) {
  constexpr int BM = 32 * NW;  // query rows per workgroup
  constexpr int BN = 32 * KB;  // keys per tile
  constexpr int TILE_BYTES = BN * D * 2;
  constexpr int KK = KS;               // contraction steps of one 32-key score block
  static_assert(KS >= 1 && KS <= D / 16, "contraction steps within the tile");
  constexpr int NS = KB * KK;          // score ops per tile
  constexpr int NV = 2 * KB * D / 32;  // PV ops per tile
  // One variable per ring slot: the compiler then knows that reading one
  // slot never overlaps the DMA into another and inserts no wait for it.
  __shared__ __attribute__((aligned(1024))) char kbuf0[TILE_BYTES];
  __shared__ __attribute__((aligned(1024))) char kbuf1[TILE_BYTES];
  __shared__ __attribute__((aligned(1024))) char vbuf0[TILE_BYTES];
  __shared__ __attribute__((aligned(1024))) char vbuf1[TILE_BYTES];
  char* const kbuf[2] = {kbuf0, kbuf1};
  char* const vbuf[2] = {vbuf0, vbuf1};
  debug_poison_lds(kbuf0, kbuf1, vbuf0, vbuf1);

  const int work = xcd_remap(blockIdx.x, total);
  const int bh = work / n_qtiles;
  const int qt = work - bh * n_qtiles;
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6, h = lane >> 5;

  // queries (and O, LSE) have Nq rows per (b, h), keys and values Nk
  const int chr = dr >> 3;  // 16-byte chunks of a row that hold data
  const int ldq = 2 * mq.ld, ldk = 2 * mk.ld, ldv = 2 * mv.ld;  // row strides in bytes
  const rsrc_t rq = make_rsrc(q + mq.head(bh, H), (unsigned)(Nq * ldq));
  const rsrc_t rk = make_rsrc(k + mk.head(bh, H), (unsigned)(Nk * ldk));
  const rsrc_t rv = make_rsrc(v + mv.head(bh, H), (unsigned)(Nk * ldv));

  // Q fragments of this wave's 32 query rows (B operands of K Q^T)
  const int qrow = qt * BM + wave * 32 + (lane & 31);
  bf16x8 qf[KK];
#pragma unroll
  for (int kk = 0; kk < KK; ++kk) qf[kk] = as_bf16x8(buffer_load16(rq, chunk_offset(qrow, 2 * kk + h, ldq, chr)));

  TileDma<D, BN, NW> dma, dmv;  // K and V tiles (the two may have different row strides)
  dma.init(wave, lane, ldk, chr);
  dmv.init(wave, lane, ldv, chr);
  RowFrag<D> kfrag;
  kfrag.init(lane);
  TrFrag<D> vfrag;
  vfrag.init(lane);

  f32x16 oacc[D / 32];
#pragma unroll
  for (int cb = 0; cb < D / 32; ++cb) oacc[cb] = zero16();
  float m_run = -INFINITY;  // running max of scaled logits, log2 units
  float l_part = 0.f;       // this lane's share of the sum of the fp32 probabilities

  const int n_kt = (Nk + BN - 1) / BN;
  dma.issue(rk, 0, ldk, kbuf[0]);
  dmv.issue(rv, 0, ldv, vbuf[0]);
  dma.issue(rk, BN, ldk, kbuf[1]);
  wait_vmem();
  __syncthreads();

  constexpr int NE = 16 * KB;  // scores per lane per tile
  // keys past the end arrive as zeros; their scores become -inf
  auto mask_ragged = [&](f32x16 (&s)[KB], int tile) {
    const int key0 = tile * BN;
    if (key0 + BN > Nk) {
#pragma unroll
      for (int kb = 0; kb < KB; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          if (key0 + kb * 32 + acc_row(r, h) >= Nk) s[kb][r] = -INFINITY;
    }
  };
  // lane-local maximum of quarter q of a tile's scores
  auto max_quarter = [&](const f32x16 (&s)[KB], int q) {
    float m = -INFINITY;
#pragma unroll
    for (int e = q * NE / 4; e < (q + 1) * NE / 4; ++e) m = fmaxf(m, s[e / 16][e % 16]);
    return m;
  };
  // fold a tile's lane-local maximum into the running max (log2 units);
  // alpha rescales what was accumulated against the old max
  float alpha = 1.f;
  bool raise = false;
  auto max_finish = [&](float mx) {
    const float m_tile = max_halves(mx) * c;
    raise = m_tile > m_run;
    const float m_new = fmaxf(m_run, m_tile);
    alpha = __builtin_amdgcn_exp2f(m_run - m_new);
    m_run = m_new;
  };

  f32x16 sa[KB], sb[KB];
#pragma unroll
  for (int i = 0; i < NS; ++i) {
    if (i % KK == 0) sa[i / KK] = zero16();
    sa[i / KK] = mfma32(lds_frag_row(kbuf[0], (i / KK) * 32 * 2 * D + kfrag.at(i % KK)), qf[i % KK], sa[i / KK]);
  }
  if (n_kt == 1) mask_ragged(sa, 0);
  max_finish(fmaxf(fmaxf(max_quarter(sa, 0), max_quarter(sa, 1)), fmaxf(max_quarter(sa, 2), max_quarter(sa, 3))));
  __syncthreads();  // kbuf[0] is refilled by the first stage

  // Stage j (parity P = j & 1, known at compile time so every LDS address is
  // a lane offset plus an immediate). On entry s holds tile j's scores and
  // m_run already covers them. One stream of NS score ops (tile j+1, into
  // sn) then NV PV ops (tile j), each with its LDS operand read two ops
  // ahead; the vector work rides along: the exponentials of tile j spread
  // over the stream (the probabilities of 16-key step t are complete two ops
  // before the PV op that uses them), this wave's DMA requests for K_{j+2}
  // and V_{j+1} on the first odd slots, and the maximum of tile j+1 in the
  // last slots. Reads K_{j+1} (kbuf[1-P]) and V_j (vbuf[P]); refills kbuf[P]
  // and vbuf[1-P].
  auto stage = [&](auto parity, auto has_next, f32x16 (&s)[KB], f32x16 (&sn)[KB], int j) {
    constexpr int P = decltype(parity)::value;
    constexpr bool NEXT = decltype(has_next)::value;
    constexpr int CPB = D / 32;  // PV ops per 16-key step
    const char* ks = kbuf[1 - P];
    const char* vs = vbuf[P];
    const float m_cur = m_run;
    float ls0 = 0.f, ls1 = 0.f;
    u32x4 pq[2 * KB];  // bf16 P^T operands, four pairs per 16-key step
    float xe[NE];
    // exponentials of the scores e with first + e*W/NE == i
    auto exp_slice = [&](auto I, auto WC) __attribute__((always_inline)) {
      constexpr int i = decltype(I)::value;
      constexpr int W = decltype(WC)::value;
      static_for<0, NE>([&](auto EC) __attribute__((always_inline)) {
        constexpr int e = decltype(EC)::value;
        if constexpr (e * W / NE == i) {
          xe[e] = __builtin_amdgcn_exp2f(__builtin_fmaf(s[e / 16][e % 16], c, -m_cur));
          if constexpr ((e & 1) != 0) {
            const bf16x2 b = {(__bf16)xe[e - 1], (__bf16)xe[e]};
            ls0 += xe[e - 1];
            ls1 += xe[e];
            pin(ls0);  // keep the exponentials in this slice
            pin(ls1);
            constexpr int pr = e / 2;
            pq[pr / 4][pr % 4] = __builtin_bit_cast(uint32_t, b);
          }
        }
      });
    };
    auto pfrag = [&](int t) { return __builtin_bit_cast(bf16x8, pq[t]); };

    if constexpr (NEXT) {
      constexpr int NOPS = NS + NV;
      constexpr int W = exp_window(NS, CPB, KB, NOPS);  // exponentials in slots 0 .. W-1
      static_assert(exp_schedule_ok(NS, CPB, KB, W), "probabilities must be ready before their PV op");
      constexpr int NDMA = 2 * decltype(dma)::PER_WAVE;
      static_assert(2 * NDMA - 1 < NOPS, "DMA requests must fit the stream");
      // score op i: key block i % KB, contraction step i / KB (the KB
      // accumulator chains are interleaved, so consecutive ops are independent)
      auto load_op = [&](int i) -> bf16x8 {
        if (i < NS) return lds_frag_row(ks, (i % KB) * 32 * 2 * D + kfrag.at(i / KB));
        const int t = i - NS;
        return vfrag.load(vs, 16 * (t / CPB), t % CPB);
      };
      float mq[4];
      bf16x8 opq[3];
      opq[0] = load_op(0);
      opq[1] = load_op(1);
      sched_fence();
      static_for<0, NOPS>([&](auto IC) __attribute__((always_inline)) {
        constexpr int i = decltype(IC)::value;
        // the ops that carry vector work run at a raised wave priority, the
        // exponentials' slots higher than the next tile's max (measured 1.4-
        // 3.6 % faster than no raise, same bits)
        if constexpr (i == 0) __builtin_amdgcn_s_setprio(2);
        if constexpr (i == W) __builtin_amdgcn_s_setprio(1);
        if constexpr (i == W + 4) __builtin_amdgcn_s_setprio(0);
        if constexpr (i + 2 < NOPS) opq[(i + 2) % 3] = load_op(i + 2);
        if constexpr (i < NS) {
          if constexpr (i / KB == 0) sn[i % KB] = zero16();
          sn[i % KB] = mfma32(opq[i % 3], qf[i / KB], sn[i % KB]);
        } else {
          constexpr int t = i - NS;
          oacc[t % CPB] = mfma32(opq[i % 3], pfrag(t / CPB), oacc[t % CPB]);
        }
        if constexpr ((i & 1) == 1 && i / 2 < NDMA) {
          constexpr int q = i / 2, PW = NDMA / 2;
          if constexpr (q < PW)
            dma.issue_one(rk, (j + 2) * BN, ldk, kbuf[P], q);
          else
            dmv.issue_one(rv, (j + 1) * BN, ldv, vbuf[1 - P], q - PW);
        }
        exp_slice(IC, std::integral_constant<int, W>{});
        if constexpr (i >= W && i < W + 4) {
          if constexpr (i == W) mask_ragged(sn, j + 1);
          mq[i - W] = max_quarter(sn, i - W);
          pin(mq[i - W]);
        }
        sched_fence();
      });
      l_part += ls0 + ls1;
      max_finish(fmaxf(fmaxf(mq[0], mq[1]), fmaxf(mq[2], mq[3])));
      l_part *= alpha;
      if (__any(raise)) {
#pragma unroll
        for (int cb = 0; cb < D / 32; ++cb)
#pragma unroll
          for (int r = 0; r < 16; ++r) oacc[cb][r] *= alpha;
      }
      wait_vmem();
      __syncthreads();
    } else {
      // last tile: all exponentials, then O^T += V^T P^T
      exp_slice(std::integral_constant<int, 0>{}, std::integral_constant<int, 1>{});
      bf16x8 vq[3];
      vq[0] = vfrag.load(vs, 0, 0);
      vq[1] = vfrag.load(vs, 16 * (1 / CPB), 1 % CPB);
      sched_fence();
#pragma unroll
      for (int i = 0; i < NV; ++i) {
        if (i + 2 < NV) vq[(i + 2) % 3] = vfrag.load(vs, 16 * ((i + 2) / CPB), (i + 2) % CPB);
        oacc[i % CPB] = mfma32(vq[i % 3], pfrag(i / CPB), oacc[i % CPB]);
        sched_fence();
      }
      l_part += ls0 + ls1;
    }
  };

  using P0 = std::integral_constant<int, 0>;
  using P1 = std::integral_constant<int, 1>;
  int j = 0;
  for (; j + 2 < n_kt; j += 2) {
    stage(P0{}, std::true_type{}, sa, sb, j);
    stage(P1{}, std::true_type{}, sb, sa, j + 1);
  }
  if (j + 1 < n_kt) {
    stage(P0{}, std::true_type{}, sa, sb, j);
    stage(P1{}, std::false_type{}, sb, sa, j + 1);
  } else {
    stage(P0{}, std::false_type{}, sa, sb, j);
  }

  // epilogue: O = O^T / l (stored transposed back to [query][d]), LSE in nats.
  const float l = sum_halves(l_part);
  if (qrow < Nq) {
    const float inv = 1.0f / l;
    float* orow = o + mo.head(bh, H) + (size_t)qrow * mo.ld;
#pragma unroll
    for (int cb = 0; cb < D / 32; ++cb)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int col = 32 * cb + 8 * g + 4 * h;  // d is a multiple of 8: four columns are all in or all out
        float4 val = make_float4(oacc[cb][4 * g] * inv, oacc[cb][4 * g + 1] * inv, oacc[cb][4 * g + 2] * inv,
                                 oacc[cb][4 * g + 3] * inv);
        if (col < dr) *reinterpret_cast<float4*>(orow + col) = val;
      }
    if (h == 0) lse[(size_t)bh * Nq + qrow] = (m_run + __log2f(l)) * kLn2;
  }
}

template <int D, int KB, int NW, int MINW, int KS = D / 16>
static hipError_t launch_fwd_v(const FwdArgs& a) {
  constexpr int BM = 32 * NW;
  const int n_qtiles = (a.Nq + BM - 1) / BM;
  const int total = a.BH * n_qtiles;
  const float c = a.scale * kLog2e;
  hipLaunchKernelGGL((attn_fwd_kernel<D, KB, NW, MINW, KS>), dim3(total), dim3(64 * NW), 0, a.stream, a.q, a.k, a.v,
                     a.o, a.lse, a.mq, a.mk, a.mv, a.mo, a.H, a.d, a.Nq, a.Nk, n_qtiles, total, c);
  return hipGetLastError();
}

// Every tile variant is instantiated explicitly: hipcc otherwise omits the
// host-side launch stub of some instantiations reached only through this
// dispatch, and the library then fails to load.
#define VITATTN_FWD_VARIANTS(X) \
  X(128, 2, 8, 2, 8) X(64, 2, 8, 2, 4) X(64, 2, 12, 3, 4) X(96, 2, 8, 2, 6) X(96, 2, 8, 2, 5) X(160, 1, 8, 2, 10)
#define VITATTN_FWD_INSTANTIATE(D, KB, NW, MINW, KS)                                                           \
  template __global__ void attn_fwd_kernel<D, KB, NW, MINW, KS>(                                              \
      const uint16_t* __restrict__, const uint16_t* __restrict__, const uint16_t* __restrict__,               \
      float* __restrict__, float* __restrict__, const Map, const Map, const Map, const Map, int, int, int, int, \
      int, int, float);
VITATTN_FWD_VARIANTS(VITATTN_FWD_INSTANTIATE)
#undef VITATTN_FWD_INSTANTIATE

// Workgroups of a forward variant resident on the current device at once (0
// if the runtime cannot say), looked up once per device.
template <int D, int KB, int NW, int MINW>
static int fwd_resident_workgroups() {
  static std::atomic<int> known[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 0;
  int n = known[dev].load(std::memory_order_relaxed);
  if (n == 0) {
    int per_cu = 0, cus = 0;
    n = -1;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, attn_fwd_kernel<D, KB, NW, MINW>, 64 * NW, 0) ==
            hipSuccess &&
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && per_cu * cus > 0)
      n = per_cu * cus;
    known[dev].store(n, std::memory_order_relaxed);
  }
  return n > 0 ? n : 0;
}

// At the narrowest tile the kernel's ~160 VGPRs fit three waves per SIMD: 12
// waves (384 queries) per workgroup share each K / V tile and hide more of
// the exponentials, ~4-6 % faster per query than 8 waves (measured at N =
// 188,416 and 1,048,576), but in coarser work items. The variant with the
// shorter estimated time (whole rounds of resident workgroups x queries per
// workgroup / that rate) is launched; each query row is computed by the
// same operations in the same order either way, so the choice changes no bit.
static hipError_t launch_fwd_64(const FwdArgs& a) {
  const int s8 = fwd_resident_workgroups<64, 2, 8, 2>(), s12 = fwd_resident_workgroups<64, 2, 12, 3>();
  if (s8 <= 0 || s12 <= 0) return launch_fwd_v<64, 2, 8, 2>(a);
  const long long t8 = (long long)a.BH * ((a.Nq + 255) / 256), t12 = (long long)a.BH * ((a.Nq + 383) / 384);
  const double c8 = (double)((t8 + s8 - 1) / s8) * 8.0, c12 = (double)((t12 + s12 - 1) / s12) * 12.0 / 1.05;
  return c12 < c8 ? launch_fwd_v<64, 2, 12, 3>(a) : launch_fwd_v<64, 2, 8, 2>(a);
}

// Tile shape per width (key blocks per tile, waves per workgroup, waves per
// SIMD): two 32-key blocks per tile and 8 waves x 32 queries, except at
// D = 160, where one key block per tile keeps the registers within budget,
// and at D = 64, where 12 waves are chosen when the grid allows (above). In
// the 96-wide tile a head dim up to 80 (ViT-10B's 72) contracts the scores
// over five 16-column steps instead of six.
hipError_t launch_fwd(const FwdArgs& a) {
  switch (tile_width(a.d)) {
    case 64: return launch_fwd_64(a);
    case 96: return a.d <= 80 ? launch_fwd_v<96, 2, 8, 2, 5>(a) : launch_fwd_v<96, 2, 8, 2>(a);
    case 128: return launch_fwd_v<128, 2, 8, 2>(a);
    default: return launch_fwd_v<160, 1, 8, 2>(a);
  }
}

}  // namespace vitattn
