// Internal launch interface between the C ABI layer and the kernels.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace vitattn {

// Where the rows of one [B][H][N][d] operand live: element strides of the
// batch, head and row dimensions (the d elements of a row are contiguous).
struct Map {
  long long sb, sh;
  int ld;
  __host__ __device__ long long head(int bh, int H) const { return (bh / H) * sb + (bh % H) * sh; }
};
inline Map dense_map(int H, int N, int d) { return Map{(long long)H * N * d, (long long)N * d, d}; }

// Tile width of the attention kernels for head dim d (a multiple of 8, at
// most 160): columns d .. D-1 of every tile are zeros.
inline int tile_width(int d) { return d <= 64 ? 64 : d <= 96 ? 96 : d <= 128 ? 128 : 160; }

struct FwdArgs {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  float* o;
  float* lse;  // [B][H][Nq], dense
  Map mq, mk, mv, mo;
  int H, BH, Nq, Nk, d;  // query rows and key rows per (b, h); d the head dim
  float scale;
  hipStream_t stream;
};

struct BwdArgs {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  const float* o;
  const uint16_t* dout;
  const float* lse;  // [B][H][Nq], dense
  float* dq;
  float* dk;
  float* dv;
  float* drow;  // workspace region 0: D = rowsum(dO o O), [BH][Nq]
  float* lse2;  // workspace region 1: LSE * log2(e), [BH][Nq]
  uint16_t* ds;  // dS mode: workspace region 2 (the dS blocks), else nullptr
  Map mq, mk, mv, mo, mg, mdq, mdk, mdv;  // mg: dout
  int H, BH, Nq, Nk, d;  // query rows and key rows per (b, h); d the head dim
  float scale;
  bool accumulate_dq;  // dq += this call's dQ instead of dq = ...
  hipStream_t stream;
};

struct MergeArgs {
  const float* o_parts;    // [P][BH][N][d]
  const float* lse_parts;  // [P][BH][N]
  float* o;                // [BH][N][d]
  float* lse;              // [BH][N]
  int P, BH, N, d;
  hipStream_t stream;
};

hipError_t launch_fwd(const FwdArgs& a);

// Workspace layout of the backward pass: two fp32 regions of region_floats
// each (D, then LSE*log2(e)), every region 256-byte aligned; in the dS mode a
// third region holds the dS blocks: 2 KB per 32 keys x 32 queries of every
// head, key blocks rounded up to the dK/dV kernel's 128 keys and query blocks
// to its 64-query tiles.
inline size_t bwd_region_floats(long long rows) { return (size_t)((rows + 63) / 64) * 64; }
inline int ds_key_blocks(int Nk) { return (Nk + 127) / 128 * 4; }
inline int ds_query_blocks(int Nq) { return (Nq + 63) / 64 * 2; }
inline size_t ds_region_bytes(long long BH, int Nq, int Nk) {
  return (size_t)BH * ds_key_blocks(Nk) * ds_query_blocks(Nq) * 2048;
}

// Backward stages; launch_bwd runs all three in order.
hipError_t launch_bwd_rowdot(const BwdArgs& a);
hipError_t launch_bwd_dkdv(const BwdArgs& a);
hipError_t launch_bwd_dq(const BwdArgs& a);  // dQ from stored dS when a.ds is set
hipError_t launch_bwd(const BwdArgs& a);
hipError_t launch_merge(const MergeArgs& a);

// Ulysses layout copies (see vitattn_ulysses.hip for the row orders)
enum { kUlyssesPack = 0, kUlyssesUnpack = 1, kUlyssesPackOut = 2, kUlyssesUnpackOut = 3 };
struct UlyssesArgs {
  const void* src;
  void* dst;
  int B, Nl, H, P, row_bytes, mode;
  hipStream_t stream;
};
hipError_t launch_ulysses(const UlyssesArgs& a);
long ulysses_blocks(int Nl, int H, int row_bytes);  // grid.x of the layout kernels

// Channel aggregation (attention of one learnable query per head over the C
// channel tokens of each of M patches); see vitattn_agg.hip.
constexpr int kAggChunkGroup = 12;  // 1 KB chunks of a [C][d] block whose loads one wave issues together
struct AggArgs {
  const uint16_t* q;     // [H][d]
  const uint16_t* k;     // [M][H][C][d]
  const uint16_t* v;     // [M][H][C][d]
  const float* o;        // [M][H][d]      (backward input)
  const uint16_t* dout;  // [M][H][d]
  float* o_out;          // forward output
  const float* lse;      // [M][H]         (backward input)
  float* lse_out;        // forward output
  float* dq;             // [H][d]
  float* dk;             // [M][H][C][d]
  float* dv;             // [M][H][C][d]
  float* partial;        // workspace: [agg_partials(M)][H][d]
  int M, H, C, d;
  float scale;
  hipStream_t stream;
};
int agg_partials(int M);  // dq partials of the backward pass
hipError_t launch_agg_fwd(const AggArgs& a);
hipError_t launch_agg_bwd(const AggArgs& a);

}  // namespace vitattn
