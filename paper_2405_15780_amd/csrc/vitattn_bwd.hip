// Backward pass of exact non-causal attention for gfx950 (FlashAttention-2's
// backward, cited by the paper in Sec. II-F): P is recomputed from Q, K and
// the saved logsumexp, never stored.
//
//   1. preprocess:  D_i = sum_c dO_ic O_ic    (HBM-bound; stored as -D_i)
//   2. dK/dV kernel: one workgroup per 128 keys (in the recompute mode 256
//      at head dims up to 64, 192 at head dims 65-80; 32 or 64 per wave, K
//      and V held in registers); streams Q, dO, LSE and D in tiles of 64
//      queries:
//        S = Q K^T, P = exp2(S*scale*log2e - LSE*log2e)
//        dV^T += dO^T P,  dP = dO V^T,  dS = P o (dP - D),  dK^T += Q^T dS
//   3. dQ kernel: one workgroup per 256 queries (or 384 at head dims up to 80;
//      32 per wave, Q and dO held in registers); streams K and V in tiles of
//      32 keys:
//        S^T = K Q^T, P^T, dP^T = V dO^T, dS^T, dQ^T += K^T dS^T
// Splitting dQ from dK/dV costs one extra recomputation of S and dP but needs
// no atomics for dQ (accumulating dQ inside the dK/dV pass would add a 4-byte
// atomic per query, column and 128-key workgroup, B H N^2 d / 128 of them,
// and fp32 atomics sustain only ~1.3 TB/s on this part). The only atomics are
// those of the dK/dV kernel's split key blocks (two fp32 adds onto zero per
// element, which commute exactly, and every whole block forms the same two
// rounded partial sums), so results are deterministic and independent of the
// grid. As in the forward pass, operands may have any batch / head / row
// strides, and a head dim d below the tile width D is padded with zero
// columns on load and cut off on store.
#include <atomic>
#include <type_traits>

#include "vitattn_common.h"
#include "vitattn_launch.h"

namespace vitattn {

// ------------------------------------------------------------------ preprocess

// Writes the two per-row statistics the backward kernels stream: -D_i =
// -sum_c dO_ic O_ic (negated, so that the dK/dV kernel can start its dP
// accumulator at it) and LSE_i * log2(e) (the logsumexp in the base-2 units
// of the kernels' exp2). Each lives in its own region of the workspace. LPR
// lanes per row take 8 columns each (lanes past the head dim add nothing).
template <int LPR>
__global__ __launch_bounds__(256) void attn_bwd_rowdot_kernel(const uint16_t* __restrict__ dout,
                                                              const float* __restrict__ o,
                                                              const float* __restrict__ lse, float* __restrict__ drow,
                                                              float* __restrict__ lse2, const Map mg, const Map mo,
                                                              int H, int N, int dr, int rows) {
  const int row = blockIdx.x * (256 / LPR) + threadIdx.x / LPR;
  const int part = threadIdx.x % LPR;
  float acc = 0.f;
  if (row < rows && part * 8 < dr) {
    const int bh = row / N, n = row - bh * N;
    const uint16_t* gp = dout + mg.head(bh, H) + (long long)n * mg.ld + part * 8;
    const float* op = o + mo.head(bh, H) + (long long)n * mo.ld + part * 8;
    const uint4 g = *reinterpret_cast<const uint4*>(gp);
    const float4 o0 = *reinterpret_cast<const float4*>(op);
    const float4 o1 = *reinterpret_cast<const float4*>(op + 4);
    const bf16x8 gb = as_bf16x8(g);
    acc = (float)gb[0] * o0.x + (float)gb[1] * o0.y + (float)gb[2] * o0.z + (float)gb[3] * o0.w +
          (float)gb[4] * o1.x + (float)gb[5] * o1.y + (float)gb[6] * o1.z + (float)gb[7] * o1.w;
  }
#pragma unroll
  for (int m = LPR / 2; m >= 1; m >>= 1) acc += __shfl_xor(acc, m, 64);
  if (row < rows && part == 0) {
    drow[row] = -acc;
    lse2[row] = lse[row] * kLog2e;
  }
}

// ------------------------------------------------------------------ dK / dV

constexpr int kDkvBQ = 64;              // queries per streamed tile
constexpr int kDkvAhead = 2;            // LDS operand reads this many matrix-core ops ahead (3 measured no better)

// Direct global -> LDS copy of a tile's row statistics: 64 floats of D and
// 64 of LSE*log2(e) (one dword per lane; rows past the end read as zeros).
// Every wave copies the same data, so that all waves issue the same number
// of loads per tile and one vmcnt bound fits them all.
__device__ __forceinline__ void stats_dma(rsrc_t rd, rsrc_t rl, int row0, float* lds_stats, int lane) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(rd, (lds_void_t*)(lds_stats), 4, (row0 + lane) * 4, 0, 0, 0);
  __builtin_amdgcn_raw_ptr_buffer_load_lds(rl, (lds_void_t*)(lds_stats + kDkvBQ), 4, (row0 + lane) * 4, 0, 0, 0);
}

// One workgroup = 2*KBW waves = 32*KBW*KPW keys of one (b, h): KBW pairs of
// waves, each pair owning KPW blocks of 32 keys (KBW = 4, KPW = 1: 8 waves,
// 128 keys; KBW = 4, KPW = 2 at the narrowest tile: 8 waves, 256 keys;
// KBW = 6, KPW = 1 in the 96-wide tile at d <= 80: 12 waves, 192 keys). The
// two waves of a pair split the roles (waves share the SIMDs round robin, so
// the vector and matrix phases of the roles interleave):
//   role P  (waves 0 .. KBW-1): holds K, accumulates dV^T.
//     S = Q K^T;  P = exp2(S*scale*log2e - LSE2);  dV^T += dO^T P;
//     writes P (bf16) to LDS for its partner.
//   role dS (waves KBW .. 2*KBW-1): holds V, accumulates dK^T, one tile behind.
//     dP = dO V^T;  dS = P o (dP - D) with the partner's P;  dK^T += Q^T dS.
// A wave with KPW key blocks reads each streamed operand from LDS once and
// feeds it to the matrix-core op of every block, and reads the row
// statistics once for all of them, so these LDS reads per matrix-core op
// shrink by a factor KPW (the P exchange stays per key block). Each key
// block's ops, and so its bits, are the same for every KPW.
// Q, dO and the row statistics stream through a ring of three LDS slots in
// tiles of 64 queries (two blocks of 32); in iteration t role P works on
// tile t and role dS on tile t-1, and tile t+1 is being fetched. Query rows
// past the end arrive as zeros and then contribute exactly nothing (P =
// exp2(0) = 1 multiplies dO = 0, and dS = P (dP - D) = 0), so the tile count
// is rounded up until the middle iterations group into threes, and every
// slot index is then a compile-time constant (LDS addresses fold into
// instruction immediates).
//
// Each wave's work per tile is one stream of 2*KPW*(KS + D/16) matrix-core
// ops whose LDS operands are read two operands ahead, in four phases (query
// blocks 0, 1; within a phase the KPW ops that share an operand are
// adjacent; the first products contract over the KS 16-column steps of d
// that hold data, D/16 or 5 for d <= 80 in the 96-wide tile):
//   1. first product of block 0 (S or dP)
//   2. first product of block 1;  vector units: P or dS of block 0
//   3. second product of block 0 (dV or dK);  vector units: block 1
//   4. second product of block 1
//
// With STORE_DS the dS waves also write every dS block they form (bf16, the
// operand of their dK product) to ds_out, for the dQ-from-dS kernel below.
// A tile's blocks are stored at the start of the wave's next tile, before
// that tile's DMA requests: loads and stores share one completion counter
// and may complete out of order with respect to each other, so a store must
// never sit between a DMA request and the wait for it.
//
// Grid balance: with one workgroup per CU, a grid that is not a whole number
// of rounds leaves CUs idle in its last round. Workgroups below n_whole each
// own a key block and every query; the key blocks after them (at most half a
// round of them) are split into two workgroups each, one per half of the
// query tiles, which add their dK and dV into rows the launch zeroed first.
template <int D, bool STORE_DS, int KBW, int KPW, int KS = D / 16>
__global__ __launch_bounds__(128 * KBW, KBW / 2) __attribute__((amdgpu_waves_per_eu(KBW / 2, KBW / 2))) void attn_bwd_dkdv_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k, const uint16_t* __restrict__ v,
    const uint16_t* __restrict__ dout, const float* __restrict__ drow, const float* __restrict__ lse2,
    float* __restrict__ dk, float* __restrict__ dv, uint16_t* __restrict__ ds_out, const Map mq, const Map mk,
    const Map mv, const Map mg, const Map mdk, const Map mdv, int H, int dr, int Nq, int Nk, int n_ktiles,
    int n_whole, float c, float scale) {
  constexpr int KK = D / 16, NCB = D / 32;
  static_assert(KS >= 1 && KS <= KK, "contraction steps within the tile");
  // operands per phase (each feeding KPW ops): first products (S or dP)
  // contract over d, second products (dV^T or dK^T) over 32 queries for each
  // of the NCB 32-column blocks of d
  constexpr int P1 = KS, P2 = KK;
  constexpr int NA = 2 * P1 + 2 * P2;  // streamed operands per tile
  constexpr int PMIN = P1 < P2 ? P1 : P2;
  // phase of streamed operand a, and the first operand of phase ph
  constexpr auto phase_of = [](int a) { return a < P1 ? 0 : a < 2 * P1 ? 1 : a < 2 * P1 + P2 ? 2 : 3; };
  constexpr auto phase_start = [](int ph) { return ph < 2 ? ph * P1 : 2 * P1 + (ph - 2) * P2; };
  constexpr int TILE_BYTES = kDkvBQ * D * 2;
  constexpr int RING = 3;
  constexpr int NWAVES = 2 * KBW;
  constexpr int BK = 32 * KBW * KPW;  // keys per workgroup
  static_assert(KPW == 1 || !STORE_DS, "stored dS blocks are laid out per wave of one key block");
  static_assert(KPW == 1 || D != 160, "the widest tile has no registers for a second key block");
  // One variable per ring slot: the compiler then knows that reading one
  // slot never overlaps the DMA into another and inserts no wait for it.
  __shared__ __attribute__((aligned(1024))) char qbuf0[TILE_BYTES];
  __shared__ __attribute__((aligned(1024))) char qbuf1[TILE_BYTES];
  __shared__ __attribute__((aligned(1024))) char qbuf2[TILE_BYTES];
  __shared__ __attribute__((aligned(1024))) char gbuf0[TILE_BYTES];
  __shared__ __attribute__((aligned(1024))) char gbuf1[TILE_BYTES];
  __shared__ __attribute__((aligned(1024))) char gbuf2[TILE_BYTES];
  __shared__ __attribute__((aligned(16))) float sbuf0[2 * kDkvBQ];  // [D | LSE2]
  __shared__ __attribute__((aligned(16))) float sbuf1[2 * kDkvBQ];
  __shared__ __attribute__((aligned(16))) float sbuf2[2 * kDkvBQ];
  static_assert(RING == 3, "one variable per slot");
  char* const qbuf[RING] = {qbuf0, qbuf1, qbuf2};
  char* const gbuf[RING] = {gbuf0, gbuf1, gbuf2};
  float* const sbuf[RING] = {sbuf0, sbuf1, sbuf2};
  // P exchange: [slot][wave pair][key block of the pair][query block]
  // [contraction step][lane] of 8 bf16. Role P writes tile t's P at the end of iteration t and role dS reads
  // it at the start of iteration t+1, so two slots (by tile parity) suffice;
  // the narrower tiles use the ring slot instead, a compile-time index. The
  // widest tile needs the two-slot form to fit in LDS.
  constexpr int XR = D == 160 ? 2 : RING;
  __shared__ __attribute__((aligned(16))) uint4 xbuf[XR][KBW][KPW][2][2][64];
  debug_poison_lds(qbuf0, qbuf1, qbuf2, gbuf0, gbuf1, gbuf2, sbuf0, sbuf1, sbuf2, xbuf);

  // this workgroup's key block (work item) and query tiles [t0, t1)
  const int n_qt_real = (Nq + kDkvBQ - 1) / kDkvBQ;
  const bool split = (int)blockIdx.x >= n_whole;
  int work, t0 = 0, t1 = n_qt_real;
  if (!split) {
    work = xcd_remap(blockIdx.x, n_whole);
  } else {
    const int part = blockIdx.x - n_whole;
    work = n_whole + (part >> 1);
    if (part & 1) t0 = n_qt_real >> 1;
    else t1 = n_qt_real >> 1;
  }
  // Every key block sums its query tiles as two partial sums split at tile
  // mid, each scaled and rounded on its own, then added: a split half adds
  // its partial onto the zeroed row; a whole block runs the tile loop twice,
  // over [0, mid) and [mid, n), storing the first partial in between and
  // adding the second to it at the end. The two fp32 adds onto zero commute,
  // so dK and dV have the same bits whether or not the grid splits the block
  // (and so for any grid shape or CU count).
  const int mid = n_qt_real >> 1;
  const bool two_part = !split && mid > 0;
  if (two_part) t1 = mid;
  const int bh = work / n_ktiles;
  const int kt = work - bh * n_ktiles;
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6, h = lane >> 5;
  const int kb = wave % KBW;
  const bool role_p = wave < KBW;

  // queries, dO and the row statistics have Nq rows per (b, h); K, V, dK, dV have Nk
  const int chr = dr >> 3;  // 16-byte chunks of a row that hold data
  const int ldq = 2 * mq.ld, ldg = 2 * mg.ld;  // row strides in bytes
  // query rows at or past qend read as zeros (the ragged end, or rows of the
  // other half or pass)
  const uint16_t* const qh = q + mq.head(bh, H);
  const uint16_t* const gh = dout + mg.head(bh, H);
  int qend = min(Nq, t1 * kDkvBQ);
  rsrc_t rq = make_rsrc(qh, (unsigned)(qend * ldq));
  rsrc_t rg = make_rsrc(gh, (unsigned)(qend * ldg));
  rsrc_t rd = make_rsrc(drow + (size_t)bh * Nq, (unsigned)qend * 4);
  rsrc_t rl = make_rsrc(lse2 + (size_t)bh * Nq, (unsigned)qend * 4);

  // held fragments (B operands, columns = this block's keys): K for role P,
  // V for role dS; this lane's key in block kp is key0 + 32 kp
  const int key0 = kt * BK + kb * 32 * KPW + (lane & 31);
  const Map& mh = role_p ? mk : mv;
  const int ldh = 2 * mh.ld;
  const rsrc_t rh = make_rsrc((role_p ? k : v) + mh.head(bh, H), (unsigned)(Nk * ldh));
  bf16x8 hf[KPW][KS];
#pragma unroll
  for (int kp = 0; kp < KPW; ++kp)
#pragma unroll
    for (int kk = 0; kk < KS; ++kk)
      hf[kp][kk] = as_bf16x8(buffer_load16(rh, chunk_offset(key0 + 32 * kp, 2 * kk + h, ldh, chr)));

  // Q and dO tiles. With STORE_DS only the four role-P waves fetch tiles, so
  // the dS waves never wait for a DMA request (and with it, for their stores).
  constexpr int DMA_WAVES = STORE_DS ? KBW : NWAVES;
  TileDma<D, kDkvBQ, DMA_WAVES> dma, dmg;
  dma.init(wave % DMA_WAVES, lane, ldq, chr);
  dmg.init(wave % DMA_WAVES, lane, ldg, chr);
  RowFrag<D> rf;
  rf.init(lane);
  TrFrag<D> tf;
  tf.init(lane);
  constexpr int DMA_PER_TILE = 2 * decltype(dma)::PER_WAVE + 2;  // loads per wave per tile

  f32x16 acc[KPW][NCB];  // dV^T (role P) or dK^T (role dS) per key block
#pragma unroll
  for (int kp = 0; kp < KPW; ++kp)
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb) acc[kp][cb] = zero16();

  // Output row of this lane's key in block kp (dV for role P, dK for role
  // dS) and the factor of its accumulator.
  auto out_row = [&](int kp) -> float* {
    const Map& mout = role_p ? mdv : mdk;
    return (role_p ? dv : dk) + mout.head(bh, H) + (size_t)(key0 + 32 * kp) * mout.ld;
  };
  const float f = role_p ? 1.f : scale;
  // Whole blocks, after their last tile below mid: store the first partial
  // (rounded like the split halves' addends) and restart the sum.
  auto store_first_part = [&]() __attribute__((always_inline)) {
#pragma unroll
    for (int kp = 0; kp < KPW; ++kp) {
      if (key0 + 32 * kp < Nk) {
        float* out = out_row(kp);
#pragma unroll
        for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
          for (int g = 0; g < 4; ++g) {
            const int col = 32 * cb + 8 * g + 4 * h;
            if (col < dr)
              *reinterpret_cast<float4*>(out + col) =
                  make_float4(acc[kp][cb][4 * g] * f, acc[kp][cb][4 * g + 1] * f, acc[kp][cb][4 * g + 2] * f,
                              acc[kp][cb][4 * g + 3] * f);
          }
      }
#pragma unroll
      for (int cb = 0; cb < NCB; ++cb) acc[kp][cb] = zero16();
    }
  };

  // Tiles are numbered from t0 in the loops below. STORE_DS: the dS operands
  // of the wave's previous tile, not yet stored (padding tiles past t1 are not).
  bf16x8 pend[2][2];
  int pend_tile = -1;
  auto flush_ds = [&]() {
    if constexpr (STORE_DS) {
      if (pend_tile >= 0 && pend_tile < t1 - t0) {
        // blocks (key block, query blocks 2t and 2t+1) of this head, 2 KB each
        const size_t nkb = (size_t)n_ktiles * KBW, nqb = 2 * (size_t)n_qt_real;
        uint16_t* dst =
            ds_out + (((size_t)bh * nkb + (size_t)kt * KBW + kb) * nqb + 2 * (size_t)(t0 + pend_tile)) * 1024;
#pragma unroll
        for (int qb = 0; qb < 2; ++qb)
#pragma unroll
          for (int ks = 0; ks < 2; ++ks)
            __builtin_nontemporal_store(pend[qb][ks],
                                        reinterpret_cast<bf16x8*>(dst + qb * 1024 + ks * 512 + lane * 8));
      }
      pend_tile = -1;
    }
  };

  auto issue_tile = [&](auto slot_tag, int t) {
    constexpr int SL = decltype(slot_tag)::value;
    const int row0 = (t0 + t) * kDkvBQ;
    dma.issue(rq, row0, ldq, qbuf[SL]);
    dmg.issue(rg, row0, ldg, gbuf[SL]);
    stats_dma(rd, rl, row0, sbuf[SL], lane);
  };

  // One tile of one role, in ring slot SL. Role P: S/P/dV; role dS: dP/dS/dK.
  // The row statistics (and role dS's P) of both query blocks are read
  // before `prefetch` requests the next tile, so that none of these LDS
  // reads has to wait for that DMA. The widest tile, and waves with more than
  // one key block, have no registers to spare for both blocks: there block
  // 1's are read into block 0's registers once block 0's vector work is done
  // (end of phase 2). Role dS starts each dP accumulator at the block's -D
  // (its 16 statistics per lane sit in the accumulator's row order), so dP -
  // D leaves the matrix cores; it then needs block 1's statistics from the
  // start and reads only block 1's P late. The widest tile keeps the
  // subtraction on the vector units.
  auto run_tile = [&](auto role_tag, auto slot_tag, int tile, auto&& prefetch) {
    constexpr bool RP = decltype(role_tag)::value;
    constexpr int SL = decltype(slot_tag)::value;
    const char* qs = qbuf[SL];
    const char* gs = gbuf[SL];
    const float* st = sbuf[SL];
    uint4(*xb)[2][2][64] = xbuf[XR == RING ? SL : (tile & 1)][kb];  // [key block][query block][step][lane]

    f32x16 m1[KPW][2];     // S (P) or dP (dS), per key block and query block
    bf16x8 ob[KPW][2][2];  // bf16 operands of P or dS [key block][query block][contraction step]
    constexpr bool LEAN = D == 160 || KPW > 1;
    constexpr bool DINIT = !RP && D != 160;      // dP accumulators start at -D
    constexpr bool LEAN_STAT = LEAN && !DINIT;   // statistics of one query block at a time
    constexpr int NSB = LEAN ? 1 : 2;  // query blocks whose P (role dS) is held at once
    constexpr int NST = LEAN_STAT ? 1 : 2;  // ... whose statistics are held at once
    float4 stat[NST][4];   // LSE2 (role P) or -D (role dS) of the block's rows
    uint4 pin4[KPW][NSB][2];  // role dS: the partner's P, as bf16 pairs

    // streamed operand a (shared by the KPW ops of one phase slot)
    auto read_a = [&](int a) -> bf16x8 {
      const int ph = phase_of(a), j = a - phase_start(ph), qb = ph & 1;
      if (ph < 2) return lds_frag_row(RP ? qs : gs, qb * 32 * 2 * D + rf.at(j));
      return tf.load(RP ? gs : qs, qb * 32 + 16 * (j / NCB), j % NCB);
    };
    auto read_stat = [&](int qb) {
#pragma unroll
      for (int g = 0; g < 4; ++g)
        stat[LEAN_STAT ? 0 : qb][g] = *reinterpret_cast<const float4*>(st + (RP ? kDkvBQ : 0) + qb * 32 + 8 * g + 4 * h);
    };
    // the 16 statistics of query block qb in accumulator order (row 8g + 4h + e
    // in element 4g + e)
    auto stat_acc = [&](int qb) {
      f32x16 v;
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const float4 t = stat[LEAN_STAT ? 0 : qb][g];
        v[4 * g] = t.x;
        v[4 * g + 1] = t.y;
        v[4 * g + 2] = t.z;
        v[4 * g + 3] = t.w;
      }
      return v;
    };
    auto read_p = [&](int qb) {
      const int sb = LEAN ? 0 : qb;
      if constexpr (!RP) {
#pragma unroll
        for (int kp = 0; kp < KPW; ++kp) {
          pin4[kp][sb][0] = xb[kp][qb][0][lane];
          pin4[kp][sb][1] = xb[kp][qb][1][lane];
        }
      }
    };
    auto valu = [&](int kp, int qb, int u, int ns) {
      // slot u of ns: rows ceil(16 u / ns) .. ceil(16 (u + 1) / ns) - 1
      constexpr int RMAX = (16 + PMIN - 1) / PMIN;
#pragma unroll
      for (int rr = 0; rr < RMAX; ++rr) {
        const int r = (u * 16 + ns - 1) / ns + rr;
        if (r >= ((u + 1) * 16 + ns - 1) / ns) break;
        const int sb = LEAN ? 0 : qb;
        const float sv = stat[LEAN_STAT ? 0 : qb][r >> 2][r & 3];
        float x;
        if constexpr (RP) {
          x = __builtin_amdgcn_exp2f(__builtin_fmaf(m1[kp][qb][r], c, -sv));
        } else {
          const unsigned w = pin4[kp][sb][r >> 3][(r & 7) >> 1];
          const float p = __uint_as_float((r & 1) ? (w & 0xffff0000u) : (w << 16));
          if constexpr (DINIT)
            x = p * m1[kp][qb][r];  // dP - D from the matrix cores
          else
            x = p * (m1[kp][qb][r] + sv);
        }
        pin(x);
        m1[kp][qb][r] = x;
        if ((r & 7) == 7) ob[kp][qb][r >> 3] = acc_to_operand(m1[kp][qb], r >> 3);
      }
    };

    if constexpr (!RP) flush_ds();  // the previous tile's dS, before this tile's DMA requests
    read_stat(0);
    read_p(0);
    if constexpr (!LEAN_STAT) read_stat(1);
    if constexpr (!LEAN) read_p(1);
    constexpr int AH = kDkvAhead;  // operand reads run AH operands ahead of their matrix-core ops
    bf16x8 aq[AH + 1];
#pragma unroll
    for (int a = 0; a < AH; ++a) aq[a] = read_a(a);
    sched_fence();
    prefetch();
    sched_fence();
    // every op index a compile-time constant (the widest tile's stream is too
    // long for the unroller's size limit, and register arrays indexed at run
    // time would live in scratch memory)
    static_for<0, NA * KPW>([&](auto IC) __attribute__((always_inline)) {
      constexpr int i = decltype(IC)::value;
      constexpr int a = i / KPW, kp = i % KPW;  // operand, key block
      constexpr int ph = phase_of(a), j = a - phase_start(ph), qb = ph & 1;
      // the two phases that carry vector work run at a raised wave priority,
      // so that their vector instructions issue ahead of the partner wave's
      // matrix-core-only phases (measured 1.7-3.3 % faster, same bits)
      if constexpr (j == 0 && kp == 0) __builtin_amdgcn_s_setprio(ph == 1 || ph == 2 ? 1 : 0);
      if constexpr (kp == 0 && a + AH < NA) aq[(a + AH) % (AH + 1)] = read_a(a + AH);
      if constexpr (ph < 2) {
        if constexpr (j == 0) {
          if constexpr (DINIT)
            m1[kp][qb] = mfma32(aq[a % (AH + 1)], hf[kp][j], stat_acc(qb));
          else
            m1[kp][qb] = mfma32(aq[a % (AH + 1)], hf[kp][j], zero16());
        } else {
          m1[kp][qb] = mfma32(aq[a % (AH + 1)], hf[kp][j], m1[kp][qb]);
        }
        if constexpr (ph == 1) valu(kp, 0, j, P1);
        if constexpr (LEAN && i == 2 * P1 * KPW - 1) {
          if constexpr (LEAN_STAT) read_stat(1);
          read_p(1);
        }
      } else {
        acc[kp][j % NCB] = mfma32(aq[a % (AH + 1)], ob[kp][qb][j / NCB], acc[kp][j % NCB]);
        if constexpr (ph == 2) valu(kp, 1, j, P2);
      }
      sched_fence();
    });
    __builtin_amdgcn_s_setprio(0);
    if constexpr (RP) {
#pragma unroll
      for (int kp = 0; kp < KPW; ++kp)
#pragma unroll
        for (int qb = 0; qb < 2; ++qb)
#pragma unroll
          for (int ks = 0; ks < 2; ++ks) xb[kp][qb][ks][lane] = __builtin_bit_cast(uint4, ob[kp][qb][ks]);
    } else if constexpr (STORE_DS) {
#pragma unroll
      for (int qb = 0; qb < 2; ++qb)
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) pend[qb][ks] = ob[0][qb][ks];
      pend_tile = tile;
    }
  };

  using S0 = std::integral_constant<int, 0>;
  using S1 = std::integral_constant<int, 1>;
  using S2 = std::integral_constant<int, 2>;
  using RoleP = std::true_type;
  using RoleDs = std::false_type;
  // Iteration t: role P on tile t (slot t % 3), role dS on tile t-1, tile t+1
  // requested into slot (t+1) % 3. Rounding the tile count to 1 mod 3 lets
  // iterations 1 .. n_pad-1 run in groups of three with fixed slots.
  int n_pad = 0;
  // Each role runs its own copy of the tile loop, so that the compiler sees
  // in the dS waves' copy that (with STORE_DS) they never have a DMA request
  // in flight, and adds no wait for one; both copies pass the same barriers.
  // End of an iteration: the fetched tile is in LDS and every wave is done
  // with the slot refilled next. With STORE_DS the dS waves issued no loads
  // and skip the wait (their stores drain in the background); a plain
  // barrier then keeps the compiler from adding a wait for every access.
  auto iteration = [&](auto role_tag, auto slot_p, auto slot_next, auto slot_ds, int t, bool run)
                       __attribute__((always_inline)) {
    constexpr bool RP = decltype(role_tag)::value;
    // tile t+1 past the end: zero rows, never read
    auto prefetch = [&]() {
      if constexpr (!STORE_DS || RP) issue_tile(slot_next, t + 1);
    };
    if constexpr (RP) {
      if (run) run_tile(RoleP{}, slot_p, t, prefetch);
      else prefetch();
    } else {
      if (run) run_tile(RoleDs{}, slot_ds, t - 1, prefetch);
      else prefetch();
    }
    if constexpr (STORE_DS) {
      if constexpr (RP) wait_vmem();
      barrier_lds();
    } else {
      wait_vmem();
      __syncthreads();
    }
  };
  auto run_role = [&](auto role_tag) __attribute__((always_inline)) {
    constexpr bool RP = decltype(role_tag)::value;
    iteration(role_tag, S0{}, S1{}, S2{}, 0, RP);
    for (int t = 1; t < n_pad; t += 3) {
      iteration(role_tag, S1{}, S2{}, S0{}, t, true);
      iteration(role_tag, S2{}, S0{}, S1{}, t + 1, true);
      iteration(role_tag, S0{}, S1{}, S2{}, t + 2, true);
    }
    // last: role dS on tile n_pad-1 (slot 0, since n_pad = 1 mod 3)
    if constexpr (!RP) {
      run_tile(RoleDs{}, S0{}, n_pad - 1, [] {});
      flush_ds();
    }
  };
  // one loop for both roles (this form keeps the default kernel's register
  // allocation; the role is a run-time branch inside each iteration)
  auto both = [&](auto slot_p, auto slot_next, auto slot_ds, int t, bool do_p, bool do_ds)
                  __attribute__((always_inline)) {
    if (role_p) {
      if (do_p) run_tile(RoleP{}, slot_p, t, [&]() { issue_tile(slot_next, t + 1); });
      else issue_tile(slot_next, t + 1);
    } else {
      if (do_ds) run_tile(RoleDs{}, slot_ds, t - 1, [&]() { issue_tile(slot_next, t + 1); });
      else issue_tile(slot_next, t + 1);
    }
    wait_vmem();
    __syncthreads();
  };
  const int n_pass = two_part ? 2 : 1;
  // Whole block between its two passes: store the first partial, then move
  // to the tiles [mid, n); every wave is done with the LDS ring and the P
  // exchange before the next pass refills them.
  auto next_pass = [&]() __attribute__((always_inline)) {
    store_first_part();
    t0 = mid;
    t1 = n_qt_real;
    qend = Nq;
    rq = make_rsrc(qh, (unsigned)(qend * ldq));
    rg = make_rsrc(gh, (unsigned)(qend * ldg));
    rd = make_rsrc(drow + (size_t)bh * Nq, (unsigned)qend * 4);
    rl = make_rsrc(lse2 + (size_t)bh * Nq, (unsigned)qend * 4);
    wait_vmem();
    __syncthreads();
  };
  auto start_pass = [&]() __attribute__((always_inline)) {
    const int n_qt = t1 - t0;
    n_pad = n_qt + (3 + 1 - n_qt % 3) % 3;
    if (!STORE_DS || role_p) issue_tile(S0{}, 0);
    wait_vmem();
    __syncthreads();
  };
  if constexpr (STORE_DS) {
    // each role runs its passes in its own branch (wave-uniform; both pass
    // the same barriers), which keeps the dS waves' loop free of the other
    // role's live values
    if (role_p) {
      for (int pass = 0; pass < n_pass; ++pass) {
        start_pass();
        run_role(RoleP{});
        if (pass + 1 < n_pass) next_pass();
      }
    } else {
      for (int pass = 0; pass < n_pass; ++pass) {
        start_pass();
        run_role(RoleDs{});
        if (pass + 1 < n_pass) next_pass();
      }
    }
  } else {
    for (int pass = 0; pass < n_pass; ++pass) {
      start_pass();
      both(S0{}, S1{}, S2{}, 0, true, false);
      for (int t = 1; t < n_pad; t += 3) {
        both(S1{}, S2{}, S0{}, t, true, true);
        both(S2{}, S0{}, S1{}, t + 1, true, true);
        both(S0{}, S1{}, S2{}, t + 2, true, true);
      }
      if (!role_p) run_tile(RoleDs{}, S0{}, n_pad - 1, [] {});
      if (pass + 1 < n_pass) next_pass();
    }
  }
  (void)DMA_PER_TILE;

  if (two_part) wait_vmem();  // the first partial's stores have completed
#pragma unroll
  for (int kp = 0; kp < KPW; ++kp) {
    if (key0 + 32 * kp >= Nk) continue;
    float* out = out_row(kp);
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int col = 32 * cb + 8 * g + 4 * h;  // d is a multiple of 8: four columns are all in or all out
        if (col < dr) {
          float x[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            x[e] = acc[kp][cb][4 * g + e] * f;
            pin(x[e]);  // rounded product, never fused into the add below
          }
          if (split) {
#pragma unroll
            for (int e = 0; e < 4; ++e) unsafeAtomicAdd(out + col + e, x[e]);
          } else if (two_part) {
            const float4 a = *reinterpret_cast<const float4*>(out + col);
            *reinterpret_cast<float4*>(out + col) = make_float4(a.x + x[0], a.y + x[1], a.z + x[2], a.w + x[3]);
          } else {
            *reinterpret_cast<float4*>(out + col) = make_float4(x[0], x[1], x[2], x[3]);
          }
        }
      }
  }
}

// Zeroes dK and dV over the key blocks of work items first .. first +
// gridDim.x/2 - 1 (rows below Nk, columns below dr), which the dK/dV kernel's
// split workgroups then add into.
__global__ __launch_bounds__(256) void zero_key_blocks_kernel(float* __restrict__ dk, float* __restrict__ dv,
                                                              const Map mdk, const Map mdv, int H, int dr, int Nk,
                                                              int n_ktiles, int first, int bk) {
  const int work = first + (blockIdx.x >> 1);
  const bool is_v = blockIdx.x & 1;
  const int bh = work / n_ktiles, kt = work - bh * n_ktiles;
  const Map& m = is_v ? mdv : mdk;
  float* base = (is_v ? dv : dk) + m.head(bh, H);
  const int c4 = dr >> 2, key0 = kt * bk, rows = min(bk, Nk - key0);
  for (int i = threadIdx.x; i < rows * c4; i += 256) {
    const int r = i / c4, c = i - r * c4;
    *reinterpret_cast<float4*>(base + (long long)(key0 + r) * m.ld + 4 * c) = make_float4(0.f, 0.f, 0.f, 0.f);
  }
}

// ------------------------------------------------------------------ dQ

// One workgroup = NW waves = 32*NW query rows of one (b, h); each wave owns
// 32 queries and keeps their Q and dO fragments (B operands), their LSE2 and
// D and the dQ^T accumulator in registers. K and V stream through a ring of
// six LDS slots in tiles of 32 keys (a barrier every second tile). Per tile j
// the wave runs
//   S^T = K_{j+1} Q^T and dP^T = V_{j+1} dO^T   (matrix cores)
//     interleaved with P^T, dS^T of tile j      (vector units)
//   dQ^T += K_j^T dS^T_j
// The tile loop is unrolled by the ring depth, so slots are compile-time
// constants and LDS addresses fold into instruction immediates. Key rows
// past the end arrive as zeros: their P is finite and they add
// K_row^T dS = 0 to dQ, so no masking is needed. S and dP contract over the
// KS 16-column steps of d that hold data (D/16, or 5 for d <= 80 in the
// 96-wide tile).
template <int D, int NW, int KS = D / 16>
__global__ __launch_bounds__(64 * NW, NW / 4) __attribute__((amdgpu_waves_per_eu(NW / 4, NW / 4))) void attn_bwd_dq_kernel(
    const uint16_t* __restrict__ q, const uint16_t* __restrict__ k, const uint16_t* __restrict__ v,
    const uint16_t* __restrict__ dout, const float* __restrict__ drow, const float* __restrict__ lse2,
    float* __restrict__ dq, const Map mq, const Map mk, const Map mv, const Map mg, const Map mdq, int H, int dr,
    int Nq, int Nk, int n_qtiles, int total, float c, float scale, int accumulate) {
  constexpr int BM = 32 * NW;
  constexpr int BN = 32;
  constexpr int KK = D / 16, NCB = D / 32;
  static_assert(KS >= 1 && KS <= KK, "contraction steps within the tile");
  constexpr int NS = 2 * KS;       // S and dP ops per tile
  constexpr int NQ = KK;           // dQ ops per tile (2 contraction steps x NCB)
  constexpr int TILE_BYTES = BN * D * 2;
  constexpr int RING = 6;
  // One variable per ring slot (no wait for reads of one slot while the DMA
  // into another is in flight).
  __shared__ __attribute__((aligned(1024))) char kbuf0[TILE_BYTES];
  __shared__ __attribute__((aligned(1024))) char kbuf1[TILE_BYTES];
  __shared__ __attribute__((aligned(1024))) char kbuf2[TILE_BYTES];
  __shared__ __attribute__((aligned(1024))) char kbuf3[TILE_BYTES];
  __shared__ __attribute__((aligned(1024))) char kbuf4[TILE_BYTES];
  __shared__ __attribute__((aligned(1024))) char kbuf5[TILE_BYTES];
  __shared__ __attribute__((aligned(1024))) char vbuf0[TILE_BYTES];
  __shared__ __attribute__((aligned(1024))) char vbuf1[TILE_BYTES];
  __shared__ __attribute__((aligned(1024))) char vbuf2[TILE_BYTES];
  __shared__ __attribute__((aligned(1024))) char vbuf3[TILE_BYTES];
  __shared__ __attribute__((aligned(1024))) char vbuf4[TILE_BYTES];
  __shared__ __attribute__((aligned(1024))) char vbuf5[TILE_BYTES];
  static_assert(RING == 6, "one variable per slot");
  char* const kbuf[RING] = {kbuf0, kbuf1, kbuf2, kbuf3, kbuf4, kbuf5};
  char* const vbuf[RING] = {vbuf0, vbuf1, vbuf2, vbuf3, vbuf4, vbuf5};
  debug_poison_lds(kbuf0, kbuf1, kbuf2, kbuf3, kbuf4, kbuf5, vbuf0, vbuf1, vbuf2, vbuf3, vbuf4, vbuf5);

  const int work = xcd_remap(blockIdx.x, total);
  const int bh = work / n_qtiles;
  const int qt = work - bh * n_qtiles;
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6, h = lane >> 5;

  // queries, dO, dQ and the row statistics have Nq rows per (b, h); K and V have Nk
  const int chr = dr >> 3;  // 16-byte chunks of a row that hold data
  const int ldq = 2 * mq.ld, ldg = 2 * mg.ld, ldk = 2 * mk.ld, ldv = 2 * mv.ld;  // row strides in bytes
  const rsrc_t rq = make_rsrc(q + mq.head(bh, H), (unsigned)(Nq * ldq));
  const rsrc_t rg = make_rsrc(dout + mg.head(bh, H), (unsigned)(Nq * ldg));
  const rsrc_t rk = make_rsrc(k + mk.head(bh, H), (unsigned)(Nk * ldk));
  const rsrc_t rv = make_rsrc(v + mv.head(bh, H), (unsigned)(Nk * ldv));

  const int qrow = qt * BM + wave * 32 + (lane & 31);
  bf16x8 qf[KS], gf[KS];
#pragma unroll
  for (int kk = 0; kk < KS; ++kk) {
    qf[kk] = as_bf16x8(buffer_load16(rq, chunk_offset(qrow, 2 * kk + h, ldq, chr)));
    gf[kk] = as_bf16x8(buffer_load16(rg, chunk_offset(qrow, 2 * kk + h, ldg, chr)));
  }
  const rsrc_t rl = make_rsrc(lse2 + (size_t)bh * Nq, (unsigned)Nq * 4);
  const rsrc_t rd = make_rsrc(drow + (size_t)bh * Nq, (unsigned)Nq * 4);
  // (the b32 buffer load returns the raw bits)
  const float l2 = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rl, qrow * 4, 0, 0));
  const float dval = -__builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rd, qrow * 4, 0, 0));  // stored -D

  TileDma<D, BN, NW> dma, dmv;  // K and V tiles
  dma.init(wave, lane, ldk, chr);
  dmv.init(wave, lane, ldv, chr);
  RowFrag<D> rf;
  rf.init(lane);
  TrFrag<D> tf;
  tf.init(lane);

  f32x16 dqacc[NCB];
#pragma unroll
  for (int cb = 0; cb < NCB; ++cb) dqacc[cb] = zero16();

  const int n_kt = (Nk + BN - 1) / BN;
  // prologue: tiles 0 .. 3 requested (tiles past the end read as zeros), scores of tile 0
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    dma.issue(rk, t * BN, ldk, kbuf[t]);
    dmv.issue(rv, t * BN, ldv, vbuf[t]);
  }
  wait_vmem();
  __syncthreads();
  f32x16 sa[2], sb[2];  // [S^T, dP^T] of the current and the next tile
#pragma unroll
  for (int i = 0; i < NS; ++i) {
    if (i % KS == 0) sa[i / KS] = zero16();
    sa[i / KS] = mfma32(lds_frag_row(i < KS ? kbuf[0] : vbuf[0], rf.at(i % KS)), i < KS ? qf[i] : gf[i - KS],
                        sa[i / KS]);
  }

  // Stage j with SL = j % RING known at compile time: P, dS of tile j (from
  // cur) and dQ of tile j (slot SL); scores of tile j+1 (slot SL+1) into nxt;
  // tile j+4 requested into the slot of tile j-2. A barrier follows every
  // second stage only: between two barriers the waves read three tiles
  // (j .. j+2 of the first stage) while three more are in flight, hence six
  // slots. The barrier after stage j waits for the requests of stage j-1 (for
  // tile j+3, read from stage j+2 on) and leaves those of stage j in flight.
  auto stage = [&](auto slot_tag, auto has_next, f32x16 (&cur)[2], f32x16 (&nxt)[2], int j) {
    constexpr int SL = decltype(slot_tag)::value;
    constexpr int NX = (SL + 1) % RING, RF = (SL + 4) % RING;
    constexpr bool NEXT = decltype(has_next)::value;
    const char* ks = kbuf[SL];
    bf16x8 dsb[2];
    // P^T and dS^T of accumulator row r of tile j
    auto row = [&](int r) {
      float p = __builtin_amdgcn_exp2f(__builtin_fmaf(cur[0][r], c, -l2));
      float g = p * (cur[1][r] - dval);
      pin(g);
      cur[1][r] = g;
      if ((r & 7) == 7) dsb[r >> 3] = acc_to_operand(cur[1], r >> 3);
    };
    if constexpr (NEXT) {
      // One stream of NS score ops (tile j+1) then NQ dQ ops (tile j), each
      // operand read one op ahead; row r of the vector work rides on op
      // r*W/16, so dS rows 8..15 are complete two ops before the dQ op that
      // first reads them.
      constexpr int NOPS = NS + NQ;
      constexpr int W = NS + NCB - 1;
      static_assert(7 * W / 16 <= NS - 2 && 15 * W / 16 <= NS + NCB - 2, "dS ready before its dQ op");
      auto load_op = [&](int i) -> bf16x8 {
        if (i < KS) return lds_frag_row(kbuf[NX], rf.at(i));
        if (i < NS) return lds_frag_row(vbuf[NX], rf.at(i - KS));
        const int t = i - NS;
        return tf.load(ks, 16 * (t / NCB), t % NCB);
      };
      bf16x8 aq[2];
      aq[0] = load_op(0);
      sched_fence();
      static_for<0, NOPS>([&](auto IC) __attribute__((always_inline)) {
        constexpr int i = decltype(IC)::value;
        // the ops that carry vector work run at a raised wave priority
        // (measured 0.3-1.1 % faster, same bits); with three waves per SIMD
        // the first half of the window runs one level higher still, so a
        // wave early in its vector work goes ahead of one late in it (3 %
        // faster at d=64, no change with two waves per SIMD)
        if constexpr (i == 0) __builtin_amdgcn_s_setprio(NW > 8 ? 2 : 1);
        if constexpr (NW > 8 && i == W / 2) __builtin_amdgcn_s_setprio(1);
        if constexpr (i == W) __builtin_amdgcn_s_setprio(0);
        if constexpr (i + 1 < NOPS) aq[(i + 1) & 1] = load_op(i + 1);
        if constexpr (i < NS) {
          if constexpr (i % KS == 0) nxt[i / KS] = zero16();
          if constexpr (i < KS)
            nxt[0] = mfma32(aq[i & 1], qf[i], nxt[0]);
          else
            nxt[1] = mfma32(aq[i & 1], gf[i - KS], nxt[1]);
        } else {
          constexpr int t = i - NS;
          dqacc[t % NCB] = mfma32(aq[i & 1], dsb[t / NCB], dqacc[t % NCB]);
        }
        if constexpr (i == 1) dma.issue(rk, (j + 4) * BN, ldk, kbuf[RF]);
        if constexpr (i == 3) dmv.issue(rv, (j + 4) * BN, ldv, vbuf[RF]);
        static_for<0, 16>([&](auto RC) __attribute__((always_inline)) {
          constexpr int r = decltype(RC)::value;
          if constexpr (r * W / 16 == i) row(r);
        });
        sched_fence();
      });
      if constexpr ((SL & 1) == 1) {
        wait_vmem_leave<2 * decltype(dma)::PER_WAVE>();
        barrier_lds();
      }
    } else {
#pragma unroll
      for (int r = 0; r < 16; ++r) row(r);
      bf16x8 aq[2];
      aq[0] = tf.load(ks, 0, 0);
      sched_fence();
#pragma unroll
      for (int i = 0; i < NQ; ++i) {
        if (i + 1 < NQ) aq[(i + 1) & 1] = tf.load(ks, 16 * ((i + 1) / NCB), (i + 1) % NCB);
        dqacc[i % NCB] = mfma32(aq[i & 1], dsb[i / NCB], dqacc[i % NCB]);
        sched_fence();
      }
    }
  };

  using S0 = std::integral_constant<int, 0>;
  using S1 = std::integral_constant<int, 1>;
  using S2 = std::integral_constant<int, 2>;
  using S3 = std::integral_constant<int, 3>;
  using S4 = std::integral_constant<int, 4>;
  using S5 = std::integral_constant<int, 5>;
  using Y = std::true_type;
  using F = std::false_type;
  // The tile count is rounded up to a multiple of the ring depth: the extra
  // tiles are all zero rows and add exactly nothing to dQ (see above), and
  // every stage then has a compile-time slot.
  const int n_iter = (n_kt + RING - 1) / RING * RING;
  int j = 0;
  for (; j + RING < n_iter; j += RING) {
    stage(S0{}, Y{}, sa, sb, j);
    stage(S1{}, Y{}, sb, sa, j + 1);
    stage(S2{}, Y{}, sa, sb, j + 2);
    stage(S3{}, Y{}, sb, sa, j + 3);
    stage(S4{}, Y{}, sa, sb, j + 4);
    stage(S5{}, Y{}, sb, sa, j + 5);
  }
  stage(S0{}, Y{}, sa, sb, j);
  stage(S1{}, Y{}, sb, sa, j + 1);
  stage(S2{}, Y{}, sa, sb, j + 2);
  stage(S3{}, Y{}, sb, sa, j + 3);
  stage(S4{}, Y{}, sa, sb, j + 4);
  stage(S5{}, F{}, sb, sa, j + 5);
  wait_vmem();  // requests past the last tile must land before this LDS is reassigned

  if (qrow < Nq) {
    float* row = dq + mdq.head(bh, H) + (size_t)qrow * mdq.ld;
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int col = 32 * cb + 8 * g + 4 * h;  // d is a multiple of 8: four columns are all in or all out
        if (col >= dr) continue;
        float4* dst = reinterpret_cast<float4*>(row + col);
        float4 val = make_float4(dqacc[cb][4 * g] * scale, dqacc[cb][4 * g + 1] * scale,
                                 dqacc[cb][4 * g + 2] * scale, dqacc[cb][4 * g + 3] * scale);
        if (accumulate) {  // this call's dQ is one key segment's share
          const float4 prev = *dst;
          val = make_float4(prev.x + val.x, prev.y + val.y, prev.z + val.z, prev.w + val.w);
        }
        *dst = val;
      }
  }
}

// ------------------------------------------------------------------ dQ from stored dS
//
// dQ = scale dS K from the dS blocks the dK/dV kernel stored: a streaming
// product with no recomputation of S and dP (2 d flops per score instead of
// 6), bound by reading dS from HBM. Block layout, one block per 32 keys x 32
// queries of one head: [bh][key block][query block][ks][lane][8] bf16 with
// ks the 16-query half and lane = 32 h + key, slot t of lane (h, key) holding
// query 16 ks + 8 (t/4) + 4 h + t%4 (the dK/dV kernel's dS operand order).
//
// One workgroup = NW waves x 32 queries of one (b, h); key tiles of 32 stream
// through a ring of six LDS slots: K (the NW waves split its DMA) and the NW
// dS blocks of the tile (each wave fetches and reads only its own block). The
// dQ^T product needs dS^T with one query per lane and 8 keys per slot group,
// the transpose of the stored order; two ds_read_b64_tr_b16 per 16 keys build
// it (lane j of a 16-lane group supplies the address of the 4 consecutive
// queries of key 16 ks + 4 h + j/4, so result lane i gets query i's entry of
// 4 consecutive keys). In the stored order, the 16 chunks (16 bytes) that a
// half-wave reads fall into only 4 of the 16 bank groups (chunk index mod 16),
// a 4-way LDS bank conflict on every read; so the DMA permutes the block's
// chunks, LDS slot s holding chunk s ^ (((s >> 5) & 3) << 2) (its own
// inverse, within the block), which spreads each half-wave's chunks over all
// 16 groups.
template <int D, int NW, int RING>
__global__ __launch_bounds__(64 * NW, 2) void attn_bwd_dq_ds_kernel(
    const uint16_t* __restrict__ k, const uint16_t* __restrict__ ds, float* __restrict__ dq, const Map mk,
    const Map mdq, int H, int dr, int Nq, int Nk, int n_qtiles, int total, int nkb, int nqb, float scale,
    int accumulate) {
  constexpr int BN = 32;
  constexpr int NCB = D / 32;
  constexpr int KTILE = BN * D * 2;  // bytes of a K tile
  constexpr int STILE = NW * 2048;   // bytes of the dS blocks of a tile
  static_assert(RING == 4 || RING == 6, "ring depth");
  __shared__ __attribute__((aligned(1024))) char kbuf0[KTILE];
  __shared__ __attribute__((aligned(1024))) char kbuf1[KTILE];
  __shared__ __attribute__((aligned(1024))) char kbuf2[KTILE];
  __shared__ __attribute__((aligned(1024))) char kbuf3[KTILE];
  __shared__ __attribute__((aligned(1024))) char kbuf4[KTILE];
  __shared__ __attribute__((aligned(1024))) char kbuf5[KTILE];
  __shared__ __attribute__((aligned(1024))) char sbuf0[STILE];
  __shared__ __attribute__((aligned(1024))) char sbuf1[STILE];
  __shared__ __attribute__((aligned(1024))) char sbuf2[STILE];
  __shared__ __attribute__((aligned(1024))) char sbuf3[STILE];
  __shared__ __attribute__((aligned(1024))) char sbuf4[STILE];
  __shared__ __attribute__((aligned(1024))) char sbuf5[STILE];
  // (a ring of four leaves the last two slot pairs unreferenced, and unallocated)
  char* const kbuf[6] = {kbuf0, kbuf1, kbuf2, kbuf3, RING > 4 ? kbuf4 : kbuf0, RING > 4 ? kbuf5 : kbuf1};
  char* const sbuf[6] = {sbuf0, sbuf1, sbuf2, sbuf3, RING > 4 ? sbuf4 : sbuf0, RING > 4 ? sbuf5 : sbuf1};
  if constexpr (RING > 4)
    debug_poison_lds(kbuf0, kbuf1, kbuf2, kbuf3, kbuf4, kbuf5, sbuf0, sbuf1, sbuf2, sbuf3, sbuf4, sbuf5);
  else
    debug_poison_lds(kbuf0, kbuf1, kbuf2, kbuf3, sbuf0, sbuf1, sbuf2, sbuf3);

  const int work = xcd_remap(blockIdx.x, total);
  const int bh = work / n_qtiles;
  const int qt = work - bh * n_qtiles;
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6, h = lane >> 5;
  const int qblock = qt * NW + wave;  // this wave's 32-query block

  const int chr = dr >> 3;
  const int ldk = 2 * mk.ld;
  const rsrc_t rk = make_rsrc(k + mk.head(bh, H), (unsigned)(Nk * ldk));
  TileDma<D, BN, NW> dma;
  dma.init(wave, lane, ldk, chr);
  TrFrag<D> tf;
  tf.init(lane);
  // dS^T operand reads: per-lane byte offsets within the wave's 2 KB block,
  // through the chunk permutation (chunk c of the stored order sits in slot
  // c ^ (m << 2), m = bits 5-6 of c; the second read of a pair, 8 chunks on,
  // flips bit 3 of the slot, hence the XOR)
  const int g = lane >> 4, j = lane & 15;
  const int c0 = (g & 1) * 64 + (j & 1) * 32 + 4 * (g >> 1) + (j >> 2);  // stored-order chunk
  const int soff_lo = 16 * (c0 ^ (((j & 1) | ((g & 1) << 1)) << 2)) + 8 * ((j >> 1) & 1);
  const int soff_hi = soff_lo ^ 128;
  // DMA: lane L of request i fills slot 64 i + L with chunk (64 i + L) ^ (m << 2)
  int ds_voff[2];
#pragma unroll
  for (int i = 0; i < 2; ++i) ds_voff[i] = 16 * ((64 * i + lane) ^ ((((lane >> 5) & 1) | (i << 1)) << 2));

  // this head's dS rows start here; key block kb's row of nqb blocks follows
  const uint16_t* ds_head = ds + (size_t)bh * nkb * nqb * 1024;
  auto issue_tile = [&](int slot_k, char* kdst, char* sdst, int t) {
    (void)slot_k;
    dma.issue(rk, t * BN, ldk, kdst);
    // the wave's own dS block of key block t (zeros past the stored blocks)
    const rsrc_t rs = make_rsrc(ds_head + (size_t)(t < nkb ? t : 0) * nqb * 1024,
                                t < nkb ? (unsigned)nqb * 2048u : 0u);
#pragma unroll
    for (int i = 0; i < 2; ++i)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (lds_void_t*)(sdst + wave * 2048 + i * 1024), 16,
                                               qblock * 2048 + ds_voff[i], 0, 0, 0);
  };
  // vector loads per wave per tile: its K share (none for the waves left
  // without one when a K tile is fewer instructions than waves) and 2 for dS
  constexpr int LOADS = decltype(dma)::PER_WAVE + 2;
  const bool k_share = decltype(dma)::ALL_ACTIVE || dma.active;

  f32x16 dqacc[NCB];
#pragma unroll
  for (int cb = 0; cb < NCB; ++cb) dqacc[cb] = zero16();

  const int n_kt = (Nk + BN - 1) / BN;
  const int n_iter = (n_kt + RING - 1) / RING * RING;  // extra tiles: zero K, add nothing
#pragma unroll
  for (int t = 0; t < RING - 1; ++t) issue_tile(t, kbuf[t], sbuf[t], t);

  // tile jj in slot SL: wait for its loads (the RING - 2 later tiles stay in
  // flight), barrier, request tile jj + RING - 1 into the slot of tile jj - 1
  // (every wave finished reading it before this barrier), then the products.
  auto stage = [&](auto slot_tag, int jj) {
    constexpr int SL = decltype(slot_tag)::value;
    constexpr int NX = (SL + RING - 1) % RING;
    if (k_share)
      wait_vmem_leave<(RING - 2) * LOADS>();
    else
      wait_vmem_leave<(RING - 2) * 2>();
    barrier_lds();
    issue_tile(NX, kbuf[NX], sbuf[NX], jj + RING - 1);
    const char* ks = kbuf[SL];
    const char* sb = sbuf[SL] + wave * 2048;
    bf16x8 dsb[2];
#pragma unroll
    for (int kh = 0; kh < 2; ++kh) {
      bf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(sb + soff_lo + kh * 256));
      bf16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(sb + soff_hi + kh * 256));
      dsb[kh][0] = lo[0]; dsb[kh][1] = lo[1]; dsb[kh][2] = lo[2]; dsb[kh][3] = lo[3];
      dsb[kh][4] = hi[0]; dsb[kh][5] = hi[1]; dsb[kh][6] = hi[2]; dsb[kh][7] = hi[3];
    }
    bf16x8 aq[2];
    aq[0] = tf.load(ks, 0, 0);
#pragma unroll
    for (int i = 0; i < 2 * NCB; ++i) {
      if (i + 1 < 2 * NCB) aq[(i + 1) & 1] = tf.load(ks, 16 * ((i + 1) / NCB), (i + 1) % NCB);
      dqacc[i % NCB] = mfma32(aq[i & 1], dsb[i / NCB], dqacc[i % NCB]);
    }
  };
  using S0 = std::integral_constant<int, 0>;
  using S1 = std::integral_constant<int, 1>;
  using S2 = std::integral_constant<int, 2>;
  using S3 = std::integral_constant<int, 3>;
  using S4 = std::integral_constant<int, 4>;
  using S5 = std::integral_constant<int, 5>;
  for (int jj = 0; jj < n_iter; jj += RING) {
    stage(S0{}, jj);
    stage(S1{}, jj + 1);
    stage(S2{}, jj + 2);
    stage(S3{}, jj + 3);
    if constexpr (RING > 4) {
      stage(S4{}, jj + 4);
      stage(S5{}, jj + 5);
    }
  }
  wait_vmem();  // requests past the last tile must land before this LDS is reassigned

  const int qrow = qblock * 32 + (lane & 31);
  if (qrow < Nq) {
    float* row = dq + mdq.head(bh, H) + (size_t)qrow * mdq.ld;
#pragma unroll
    for (int cb = 0; cb < NCB; ++cb)
#pragma unroll
      for (int gg = 0; gg < 4; ++gg) {
        const int col = 32 * cb + 8 * gg + 4 * h;  // d is a multiple of 8: four columns are all in or all out
        if (col >= dr) continue;
        float4* dst = reinterpret_cast<float4*>(row + col);
        float4 val = make_float4(dqacc[cb][4 * gg] * scale, dqacc[cb][4 * gg + 1] * scale,
                                 dqacc[cb][4 * gg + 2] * scale, dqacc[cb][4 * gg + 3] * scale);
        if (accumulate) {
          const float4 prev = *dst;
          val = make_float4(prev.x + val.x, prev.y + val.y, prev.z + val.z, prev.w + val.w);
        }
        *dst = val;
      }
  }
}

// ------------------------------------------------------------------ launch

template <int LPR>
static hipError_t rowdot_l(const BwdArgs& a) {
  const int rows = a.BH * a.Nq;
  constexpr int rows_per_block = 256 / LPR;
  hipLaunchKernelGGL(attn_bwd_rowdot_kernel<LPR>, dim3((unsigned)((rows + rows_per_block - 1) / rows_per_block)),
                     dim3(256), 0, a.stream, a.dout, a.o, a.lse, a.drow, a.lse2, a.mg, a.mo, a.H, a.Nq, a.d, rows);
  return hipGetLastError();
}

// Workgroups of the dK/dV kernel resident on the current device at once
// (0 if the runtime cannot say), looked up once per device.
template <int D, bool STORE_DS, int KBW, int KPW, int KS>
static int dkdv_resident_workgroups() {
  static std::atomic<int> known[64];  // per device ordinal; 0 = not looked up, -1 = unknown
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 0;
  int n = known[dev].load(std::memory_order_relaxed);
  if (n == 0) {
    int per_cu = 0, cus = 0;
    n = -1;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, attn_bwd_dkdv_kernel<D, STORE_DS, KBW, KPW, KS>,
                                                     128 * KBW, 0) == hipSuccess &&
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && per_cu * cus > 0)
      n = per_cu * cus;
    known[dev].store(n, std::memory_order_relaxed);
  }
  return n > 0 ? n : 0;
}

template <int D, bool STORE_DS, int KBW, int KPW, int KS = D / 16>
static hipError_t dkdv_s(const BwdArgs& a) {
  constexpr int BK = 32 * KBW * KPW;
  const int n_kt = (a.Nk + BK - 1) / BK;
  const int total = a.BH * n_kt;
  // A last round at most half full is split in two halves of the query range
  // (when there are two query tiles to split), so that it takes half as long.
  const int slots = dkdv_resident_workgroups<D, STORE_DS, KBW, KPW, KS>();
  const int tail = slots > 0 ? total % slots : 0;
  int n_whole = total;
  if (tail > 0 && 2 * tail <= slots && (a.Nq + kDkvBQ - 1) / kDkvBQ >= 2) {
    n_whole = total - tail;
    hipLaunchKernelGGL(zero_key_blocks_kernel, dim3(2 * tail), dim3(256), 0, a.stream, a.dk, a.dv, a.mdk, a.mdv, a.H,
                       a.d, a.Nk, n_kt, n_whole, BK);
  }
  const int grid = n_whole + 2 * (total - n_whole);
  hipLaunchKernelGGL((attn_bwd_dkdv_kernel<D, STORE_DS, KBW, KPW, KS>), dim3(grid), dim3(64 * 2 * KBW), 0, a.stream, a.q,
                     a.k, a.v, a.dout, a.drow, a.lse2, a.dk, a.dv, a.ds, a.mq, a.mk, a.mv, a.mg, a.mdk, a.mdv, a.H,
                     a.d, a.Nq, a.Nk, n_kt, n_whole, a.scale * kLog2e, a.scale);
  return hipGetLastError();
}
// Four pairs of waves per workgroup, except where noted. At the narrowest
// tile in the recompute mode each wave holds two 32-key blocks (222 VGPRs,
// two waves per SIMD, 256 keys per workgroup), so every operand it reads
// from LDS feeds two matrix-core ops and every Q / dO tile it streams serves
// twice the keys: 8 % faster than six one-block pairs at three waves per
// SIMD (B=4, H=1, N=188,416, d=64), with the same bits. At the wider tiles
// two blocks per wave leave room for one wave per SIMD only, which measured
// 5 % slower at d=128 and no faster at d=96. In the 96-wide tile a head dim
// up to 80 contracts S and dP over five 16-column steps instead of six, and
// the recompute mode then fits three waves per SIMD (168 VGPRs, two values
// spilled outside the tile loop): six pairs, 192 keys per workgroup, 4-5 %
// faster at d=72 on large grids, with the same bits. The dS mode keeps four
// pairs of one-block waves (its stored dS blocks are laid out per 128 keys).
template <int D>
static hipError_t dkdv_d(const BwdArgs& a) {
  if constexpr (D == 96) {
    if (a.d <= 80) return a.ds != nullptr ? dkdv_s<96, true, 4, 1, 5>(a) : dkdv_s<96, false, 6, 1, 5>(a);
  }
  if (a.ds != nullptr) return dkdv_s<D, true, 4, 1>(a);
  return dkdv_s<D, false, 4, D == 64 ? 2 : 1>(a);
}

#define VITATTN_DKDV_INSTANTIATE(D, S, KBW, KPW, KS)                                                           \
  template __global__ void attn_bwd_dkdv_kernel<D, S, KBW, KPW, KS>(                                          \
      const uint16_t* __restrict__, const uint16_t* __restrict__, const uint16_t* __restrict__,               \
      const uint16_t* __restrict__, const float* __restrict__, const float* __restrict__, float* __restrict__, \
      float* __restrict__, uint16_t* __restrict__, const Map, const Map, const Map, const Map, const Map,      \
      const Map, int, int, int, int, int, int, float, float);
VITATTN_DKDV_INSTANTIATE(128, false, 4, 1, 8)
VITATTN_DKDV_INSTANTIATE(64, false, 4, 2, 4)
VITATTN_DKDV_INSTANTIATE(96, false, 4, 1, 6)
VITATTN_DKDV_INSTANTIATE(96, false, 6, 1, 5)
VITATTN_DKDV_INSTANTIATE(160, false, 4, 1, 10)
VITATTN_DKDV_INSTANTIATE(128, true, 4, 1, 8)
VITATTN_DKDV_INSTANTIATE(64, true, 4, 1, 4)
VITATTN_DKDV_INSTANTIATE(96, true, 4, 1, 6)
VITATTN_DKDV_INSTANTIATE(96, true, 4, 1, 5)
VITATTN_DKDV_INSTANTIATE(160, true, 4, 1, 10)
#undef VITATTN_DKDV_INSTANTIATE

template <int D, int NW, int RING>
static hipError_t dq_ds_v(const BwdArgs& a) {
  const int n_qt = (a.Nq + 32 * NW - 1) / (32 * NW);
  const int total = a.BH * n_qt;
  hipLaunchKernelGGL((attn_bwd_dq_ds_kernel<D, NW, RING>), dim3(total), dim3(64 * NW), 0, a.stream, a.k, a.ds, a.dq,
                     a.mk, a.mdq, a.H, a.d, a.Nq, a.Nk, n_qt, total, ds_key_blocks(a.Nk), ds_query_blocks(a.Nq),
                     a.scale, a.accumulate_dq ? 1 : 0);
  return hipGetLastError();
}
// 8 waves and a six-slot ring measured best (6.1 TB/s at N = 188,416 against
// 4.9 for 4 waves with two workgroups per CU and 6.0 for a four-slot ring)
template <int D>
static hipError_t dq_ds_d(const BwdArgs& a) {
  return dq_ds_v<D, 8, 6>(a);
}

#define VITATTN_DQDS_INSTANTIATE(D, NW, R)                                                                    \
  template __global__ void attn_bwd_dq_ds_kernel<D, NW, R>(                                                   \
      const uint16_t* __restrict__, const uint16_t* __restrict__, float* __restrict__, const Map, const Map, int, \
      int, int, int, int, int, int, int, float, int);
VITATTN_DQDS_INSTANTIATE(64, 8, 6)
VITATTN_DQDS_INSTANTIATE(96, 8, 6)
VITATTN_DQDS_INSTANTIATE(128, 8, 6)
VITATTN_DQDS_INSTANTIATE(160, 8, 6)
#undef VITATTN_DQDS_INSTANTIATE

template <int D, int NW, int KS = D / 16>
static hipError_t dq_v(const BwdArgs& a) {
  const int n_qt = (a.Nq + 32 * NW - 1) / (32 * NW);
  const int total = a.BH * n_qt;
  hipLaunchKernelGGL((attn_bwd_dq_kernel<D, NW, KS>), dim3(total), dim3(64 * NW), 0, a.stream, a.q, a.k, a.v, a.dout,
                     a.drow, a.lse2, a.dq, a.mq, a.mk, a.mv, a.mg, a.mdq, a.H, a.d, a.Nq, a.Nk, n_qt, total,
                     a.scale * kLog2e, a.scale, a.accumulate_dq ? 1 : 0);
  return hipGetLastError();
}

#define VITATTN_DQ_INSTANTIATE(D, NW, KS)                                                                      \
  template __global__ void attn_bwd_dq_kernel<D, NW, KS>(                                                     \
      const uint16_t* __restrict__, const uint16_t* __restrict__, const uint16_t* __restrict__,               \
      const uint16_t* __restrict__, const float* __restrict__, const float* __restrict__, float* __restrict__, \
      const Map, const Map, const Map, const Map, const Map, int, int, int, int, int, int, float, float, int);
VITATTN_DQ_INSTANTIATE(128, 8, 8)
VITATTN_DQ_INSTANTIATE(64, 8, 4)
VITATTN_DQ_INSTANTIATE(64, 12, 4)
VITATTN_DQ_INSTANTIATE(96, 8, 6)
VITATTN_DQ_INSTANTIATE(96, 8, 5)
VITATTN_DQ_INSTANTIATE(96, 12, 5)
VITATTN_DQ_INSTANTIATE(160, 8, 10)
#undef VITATTN_DQ_INSTANTIATE

hipError_t launch_bwd_rowdot(const BwdArgs& a) {
  const int chunks = a.d / 8;
  return chunks <= 8 ? rowdot_l<8>(a) : chunks <= 16 ? rowdot_l<16>(a) : rowdot_l<32>(a);
}
hipError_t launch_bwd_dkdv(const BwdArgs& a) {
  switch (tile_width(a.d)) {
    case 64: return dkdv_d<64>(a);
    case 96: return dkdv_d<96>(a);
    case 128: return dkdv_d<128>(a);
    default: return dkdv_d<160>(a);
  }
}
hipError_t launch_bwd_dq_ds(const BwdArgs& a) {
  switch (tile_width(a.d)) {
    case 64: return dq_ds_d<64>(a);
    case 96: return dq_ds_d<96>(a);
    case 128: return dq_ds_d<128>(a);
    default: return dq_ds_d<160>(a);
  }
}
// Workgroups of a dQ kernel variant resident on the current device at once
// (0 if the runtime cannot say), looked up once per device.
template <int D, int NW, int KS>
static int dq_resident_workgroups() {
  static std::atomic<int> known[64];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 0;
  int n = known[dev].load(std::memory_order_relaxed);
  if (n == 0) {
    int per_cu = 0, cus = 0;
    n = -1;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, attn_bwd_dq_kernel<D, NW, KS>, 64 * NW, 0) == hipSuccess &&
        hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && per_cu * cus > 0)
      n = per_cu * cus;
    known[dev].store(n, std::memory_order_relaxed);
  }
  return n > 0 ? n : 0;
}

// At the narrowest tile (168 VGPRs, three values spilled and reloaded only
// after the tile loop) and at D = 96 with five contraction steps (168, one
// 16-byte operand spilled and reloaded three times per six tiles) the dQ
// kernel fits three waves per SIMD: 12 waves (384 queries) per workgroup share
// each K / V tile, faster per query than 8 waves (~6 % at D = 64, B=4, H=1, N=188,416;
// ~4.5 % at d = 72, B=1, H=2-3, N=50,001-188,416), but in coarser work items.
// The variant with the shorter estimated time (whole rounds of resident
// workgroups x queries per workgroup / that rate) is launched; both compute
// every dQ row with the same operations in the same order, so the choice
// changes no bit.
template <int D, int KS>
static hipError_t dq_8_or_12(const BwdArgs& a, double rate12) {
  const int s8 = dq_resident_workgroups<D, 8, KS>(), s12 = dq_resident_workgroups<D, 12, KS>();
  if (s8 <= 0 || s12 <= 0) return dq_v<D, 8, KS>(a);
  const long long t8 = (long long)a.BH * ((a.Nq + 255) / 256), t12 = (long long)a.BH * ((a.Nq + 383) / 384);
  const double c8 = (double)((t8 + s8 - 1) / s8) * 8.0, c12 = (double)((t12 + s12 - 1) / s12) * 12.0 / rate12;
  return c12 < c8 ? dq_v<D, 12, KS>(a) : dq_v<D, 8, KS>(a);
}

hipError_t launch_bwd_dq(const BwdArgs& a) {
  if (a.ds != nullptr) return launch_bwd_dq_ds(a);
  switch (tile_width(a.d)) {
    case 64: return dq_8_or_12<64, 4>(a, 1.06);
    case 96: return a.d <= 80 ? dq_8_or_12<96, 5>(a, 1.045) : dq_v<96, 8>(a);  // d <= 80: five contraction steps
    case 128: return dq_v<128, 8>(a);
    default: return dq_v<160, 8>(a);
  }
}

hipError_t launch_bwd(const BwdArgs& a) {
  hipError_t e = launch_bwd_rowdot(a);
  if (e == hipSuccess) e = launch_bwd_dkdv(a);
  if (e == hipSuccess) e = launch_bwd_dq(a);
  return e;
}

}  // namespace vitattn
