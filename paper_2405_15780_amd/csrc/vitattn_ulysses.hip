// Data layouts around DeepSpeed-Ulysses' all-to-all (the paper's best
// sequence-parallel scheme: Sec. II "Sequence Parallel", two all-to-alls per
// attention in each pass, Sec. V). Rank r holds tokens r*Nl .. (r+1)*Nl-1 of
// all H heads; attention needs the full sequence of Hl = H/P heads. Rows are
// opaque blocks of row_bytes (a multiple of 16), so bf16 Q/K/V and fp32
// outputs use the same kernel. Three row orders appear:
//   A  sequence-major   [B][Nl][H]        row (b*Nl + i)*H + p*Hl + j
//   C  per destination  [P][B][Hl][Nl]    row ((p*B + b)*Hl + j)*Nl + i
//   U  attention layout [B][Hl][P*Nl]     row (b*Hl + j)*(P*Nl) + p*Nl + i
// pack: A -> C (send buffer), unpack: C -> U (after the all-to-all, recv
// chunk p came from rank p), pack_out: U -> C, unpack_out: C -> A.
// Pure copies, bound by HBM bandwidth; one 16-byte vector per thread. A
// block copies 256 vectors of consecutive tokens of one head, and consecutive
// blocks take consecutive heads of the same tokens, so that the blocks in
// flight together sweep whole [H][row] token records of the sequence-major
// side instead of one row out of every H.
#include "vitattn_common.h"
#include "vitattn_launch.h"

namespace vitattn {

template <int MODE>
__global__ __launch_bounds__(256) void ulysses_layout_kernel(const uint4* __restrict__ src, uint4* __restrict__ dst,
                                                             int B, int Nl, int H, int P, int vpr) {
  const int hh = blockIdx.x % H;  // global head p*Hl + j
  const int idx = (blockIdx.x / H) * 256 + threadIdx.x;
  if (idx >= Nl * vpr) return;
  const int i = idx / vpr, v = idx - (idx / vpr) * vpr;
  const int Hl = H / P;
  const int p = hh / Hl, j = hh - (hh / Hl) * Hl;
  const int b = blockIdx.y;
  const long rowA = ((long)b * Nl + i) * H + hh;
  const long rowC = (((long)p * B + b) * Hl + j) * Nl + i;
  const long rowU = ((long)b * Hl + j) * ((long)P * Nl) + (long)p * Nl + i;
  long rs, rd;
  if constexpr (MODE == kUlyssesPack) {
    rs = rowA, rd = rowC;
  } else if constexpr (MODE == kUlyssesUnpack) {
    rs = rowC, rd = rowU;
  } else if constexpr (MODE == kUlyssesPackOut) {
    rs = rowU, rd = rowC;
  } else {
    rs = rowC, rd = rowA;
  }
  dst[rd * vpr + v] = src[rs * vpr + v];
}

long ulysses_blocks(int Nl, int H, int row_bytes) { return ((long)Nl * (row_bytes / 16) + 255) / 256 * H; }

template <int MODE>
static hipError_t layout_m(const UlyssesArgs& a) {
  const int vpr = a.row_bytes / 16;
  const dim3 grid((unsigned)ulysses_blocks(a.Nl, a.H, a.row_bytes), (unsigned)a.B);
  hipLaunchKernelGGL(ulysses_layout_kernel<MODE>, grid, dim3(256), 0, a.stream, static_cast<const uint4*>(a.src),
                     static_cast<uint4*>(a.dst), a.B, a.Nl, a.H, a.P, vpr);
  return hipGetLastError();
}

template __global__ void ulysses_layout_kernel<kUlyssesPack>(const uint4* __restrict__, uint4* __restrict__, int,
                                                             int, int, int, int);
template __global__ void ulysses_layout_kernel<kUlyssesUnpack>(const uint4* __restrict__, uint4* __restrict__, int,
                                                               int, int, int, int);
template __global__ void ulysses_layout_kernel<kUlyssesPackOut>(const uint4* __restrict__, uint4* __restrict__, int,
                                                                int, int, int, int);
template __global__ void ulysses_layout_kernel<kUlyssesUnpackOut>(const uint4* __restrict__, uint4* __restrict__,
                                                                  int, int, int, int, int);

hipError_t launch_ulysses(const UlyssesArgs& a) {
  switch (a.mode) {
    case kUlyssesPack: return layout_m<kUlyssesPack>(a);
    case kUlyssesUnpack: return layout_m<kUlyssesUnpack>(a);
    case kUlyssesPackOut: return layout_m<kUlyssesPackOut>(a);
    default: return layout_m<kUlyssesUnpackOut>(a);
  }
}

}  // namespace vitattn
