// C ABI of the attention library: argument validation, workspace sizing and
// status codes. Validation runs before any HIP call, so a rejected call has
// launched nothing and written nothing, and works without a GPU.
#include <math.h>
#include <stdint.h>
#include <stdlib.h>

#include <exception>
#include <mutex>

#include "../../include/vitattn.h"
#include "vitattn_launch.h"

#define VITATTN_VERSION "0.3.0"

namespace {

bool aligned16(const void* p) { return p != nullptr && (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// head dims of the attention kernels: multiples of 8 (16-byte rows) up to 160
bool head_dim_ok(int d) { return d >= 8 && d <= 160 && d % 8 == 0; }

// row counts: row indices and grid sizes are 32-bit, so B*H*N must fit in an
// int; per-head byte offsets of a dense bf16 operand (plus the padding rows of
// the last tiles) must fit in 31 bits
int check_rows(int B, int H, int N, int d) {
  if (B < 1 || H < 1 || N < 1) return VITATTN_E_INVAL;
  if ((long long)B * H * N > 0x7fffffffLL) return VITATTN_E_INVAL;
  if ((long long)(N + 256) * d * 2 > 0x7fffffffLL) return VITATTN_E_INVAL;
  return VITATTN_OK;
}

int check_sizes(int B, int H, int N, int d) {
  if (B < 1 || H < 1 || N < 1) return VITATTN_E_INVAL;
  if (!head_dim_ok(d)) return VITATTN_E_UNSUPPORTED;
  return check_rows(B, H, N, d);
}

bool scale_ok(float s) { return isfinite(s) && s > 0.f; }

// Every launch must stay below 2^32 work-items (a dispatch's grid size is
// 32-bit; a larger one would fail at launch, after the call's earlier
// kernels had run). The forward and dQ kernels run 2 per query row plus the
// padding of each head's last workgroup (up to 383 rows), the dK/dV kernel
// up to 4 per key row plus its padding (up to 191 rows per head) and the
// split workgroups of at most half a round (one per CU, 768 work-items
// each), the row-dot pass 8, 16 or 32 per row (head dims up to 64, 128,
// 160) and the merge d/4 per row. These bounds bind only at head dims of 16
// or less; wider rows run out of memory first.
constexpr long long kMaxWorkItems = 1LL << 32;
bool fwd_items_ok(int B, int H, int Nq) { return 2LL * B * H * (Nq + 383LL) < kMaxWorkItems; }
bool bwd_items_ok(int B, int H, int Nq, int Nk, int d) {
  const long long bh = (long long)B * H, lpr = d <= 64 ? 8 : d <= 128 ? 16 : 32;
  return fwd_items_ok(B, H, Nq) && 4 * bh * (Nk + 191LL) + (1LL << 19) < kMaxWorkItems &&
         bh * Nq * lpr + 256 < kMaxWorkItems;
}
bool merge_items_ok(int B, int H, int N, int d) { return (long long)B * H * N * (d / 4) + 256 < kMaxWorkItems; }

// key rows obey the same limits as query rows
int check_sizes_kv(int B, int H, int Nq, int Nk, int d) {
  const int st = check_sizes(B, H, Nq, d);
  return st != VITATTN_OK ? st : check_sizes(B, H, Nk, d);
}

// One operand's strides (elements). Rows must be 16-byte aligned and must not
// overlap (row >= d); every stride is non-negative and a multiple of
// 16 / elem_bytes elements. Operands read through buffer resources (the bf16
// inputs) must keep (N + 256) rows within 31-bit byte offsets. An output must
// not overlap itself: sorted by stride, each dimension must step past the
// span of the smaller ones. Inputs may repeat heads or batches (stride 0).
int check_map(const vitattn_strides& m, int B, int H, int N, int d, int elem_bytes, bool output) {
  const long long unit = 16 / elem_bytes;
  if (m.batch < 0 || m.head < 0 || m.row < d) return VITATTN_E_INVAL;
  if (m.batch % unit != 0 || m.head % unit != 0 || m.row % unit != 0) return VITATTN_E_INVAL;
  if (m.row > 0x7fffffffLL) return VITATTN_E_INVAL;
  if (elem_bytes == 2 && (long long)(N + 256) * m.row * 2 > 0x7fffffffLL) return VITATTN_E_INVAL;
  // the largest element offset must fit comfortably in 64 bits
  if ((double)(B - 1) * m.batch + (double)(H - 1) * m.head + (double)N * m.row > 4.0e18) return VITATTN_E_INVAL;
  if (output) {
    long long size[3] = {B, H, N}, stride[3] = {m.batch, m.head, m.row};
    int idx[3] = {0, 1, 2};
    for (int i = 0; i < 3; ++i)  // sort the three dimensions by stride
      for (int j = i + 1; j < 3; ++j)
        if (stride[idx[j]] < stride[idx[i]]) {
          const int t = idx[i];
          idx[i] = idx[j];
          idx[j] = t;
        }
    long long span = d;  // elements covered by the dimensions taken so far (a row first)
    for (int i = 0; i < 3; ++i) {
      const int x = idx[i];
      if (size[x] == 1) continue;
      if (stride[x] < span) return VITATTN_E_INVAL;
      span += (size[x] - 1) * stride[x];
    }
  }
  return VITATTN_OK;
}

vitattn::Map to_map(const vitattn_strides& m) { return vitattn::Map{m.batch, m.head, (int)m.row}; }
vitattn_strides dense(int H, int N, int d) {
  vitattn_strides m;
  m.batch = (long long)H * N * d;
  m.head = (long long)N * d;
  m.row = d;
  return m;
}

}  // namespace

extern "C" {

const char* vitattn_status_str(int status) {
  switch (status) {
    case VITATTN_OK: return "VITATTN_OK";
    case VITATTN_E_INVAL: return "VITATTN_E_INVAL: invalid argument";
    case VITATTN_E_UNSUPPORTED: return "VITATTN_E_UNSUPPORTED: unsupported head dim";
    case VITATTN_E_WORKSPACE: return "VITATTN_E_WORKSPACE: workspace missing or too small";
    case VITATTN_E_HIP: return "VITATTN_E_HIP: HIP runtime error at launch";
    case VITATTN_E_INTERNAL: return "VITATTN_E_INTERNAL: internal error";
    case VITATTN_E_TOO_LARGE:
      return "VITATTN_E_TOO_LARGE: B*H*N exceeds VITATTN_NOALLOC_MAX_ROWS, the static scratch of vitattn_bwd_noalloc";
    default: return "VITATTN: unknown status";
  }
}

const char* vitattn_version(void) { return VITATTN_VERSION; }

size_t vitattn_bwd_workspace_bytes(int B, int H, int N, int d) {
  if (check_sizes(B, H, N, d) != VITATTN_OK) return 0;
  return 2 * vitattn::bwd_region_floats((long long)B * H * N) * sizeof(float);
}

// the dS region's 32-query block rows must stay within 31-bit buffer offsets
static bool ds_mode_ok(int Nq) { return (long long)vitattn::ds_query_blocks(Nq) * 2048 <= 0x7fffffffLL; }

size_t vitattn_bwd_workspace_bytes_kv(int B, int H, int Nq, int Nk, int d, int flags) {
  if (check_sizes_kv(B, H, Nq, Nk, d) != VITATTN_OK) return 0;
  if ((flags & ~(VITATTN_BWD_ACCUMULATE_DQ | VITATTN_BWD_STORE_DS)) != 0) return 0;
  size_t bytes = vitattn_bwd_workspace_bytes(B, H, Nq, d);
  if (flags & VITATTN_BWD_STORE_DS) {
    if (!ds_mode_ok(Nq)) return 0;
    bytes += vitattn::ds_region_bytes((long long)B * H, Nq, Nk);
  }
  return bytes;
}

int vitattn_fwd(const void* q, const void* k, const void* v, float* o, float* lse, int B, int H, int N, int d,
                float scale, void* stream) {
  return vitattn_fwd_kv(q, k, v, o, lse, B, H, N, N, d, scale, stream);
}

int vitattn_fwd_kv(const void* q, const void* k, const void* v, float* o, float* lse, int B, int H, int Nq, int Nk,
                   int d, float scale, void* stream) {
  return vitattn_fwd_strided(q, dense(H, Nq, d), k, dense(H, Nk, d), v, dense(H, Nk, d), o, dense(H, Nq, d), lse, B,
                             H, Nq, Nk, d, scale, stream);
}

int vitattn_fwd_strided(const void* q, vitattn_strides sq, const void* k, vitattn_strides sk, const void* v,
                        vitattn_strides sv, float* o, vitattn_strides so, float* lse, int B, int H, int Nq, int Nk,
                        int d, float scale, void* stream) {
  try {
    int st = check_sizes_kv(B, H, Nq, Nk, d);
    if (st != VITATTN_OK) return st;
    if (!fwd_items_ok(B, H, Nq)) return VITATTN_E_INVAL;
    if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(o) || !aligned16(lse))
      return VITATTN_E_INVAL;
    if (!scale_ok(scale)) return VITATTN_E_INVAL;
    if (check_map(sq, B, H, Nq, d, 2, false) || check_map(sk, B, H, Nk, d, 2, false) ||
        check_map(sv, B, H, Nk, d, 2, false) || check_map(so, B, H, Nq, d, 4, true))
      return VITATTN_E_INVAL;
    vitattn::FwdArgs a;
    a.q = static_cast<const uint16_t*>(q);
    a.k = static_cast<const uint16_t*>(k);
    a.v = static_cast<const uint16_t*>(v);
    a.o = o;
    a.lse = lse;
    a.mq = to_map(sq);
    a.mk = to_map(sk);
    a.mv = to_map(sv);
    a.mo = to_map(so);
    a.H = H;
    a.BH = B * H;
    a.Nq = Nq;
    a.Nk = Nk;
    a.d = d;
    a.scale = scale;
    a.stream = static_cast<hipStream_t>(stream);
    return vitattn::launch_fwd(a) == hipSuccess ? VITATTN_OK : VITATTN_E_HIP;
  } catch (...) {
    return VITATTN_E_INTERNAL;
  }
}

static int check_workspace(const void* ws, size_t bytes, int B, int H, int N, int d) {
  if (ws == nullptr || (reinterpret_cast<uintptr_t>(ws) & 15u) != 0 ||
      bytes < vitattn_bwd_workspace_bytes(B, H, N, d))
    return VITATTN_E_WORKSPACE;
  return VITATTN_OK;
}

// Arguments of the backward kernels; operands without strides given are dense.
static vitattn::BwdArgs bwd_args(const void* q, const void* k, const void* v, const float* o, const void* dout,
                                 const float* lse, float* dq, float* dk, float* dv, int B, int H, int Nq, int Nk,
                                 int d, float scale, bool accumulate_dq, const void* workspace, void* stream) {
  vitattn::BwdArgs a;
  a.q = static_cast<const uint16_t*>(q);
  a.k = static_cast<const uint16_t*>(k);
  a.v = static_cast<const uint16_t*>(v);
  a.o = o;
  a.dout = static_cast<const uint16_t*>(dout);
  a.lse = lse;
  a.dq = dq;
  a.dk = dk;
  a.dv = dv;
  a.drow = static_cast<float*>(const_cast<void*>(workspace));
  a.lse2 = a.drow + vitattn::bwd_region_floats((long long)B * H * Nq);
  a.ds = nullptr;
  a.mq = a.mo = a.mg = a.mdq = to_map(dense(H, Nq, d));
  a.mk = a.mv = a.mdk = a.mdv = to_map(dense(H, Nk, d));
  a.H = H;
  a.BH = B * H;
  a.Nq = Nq;
  a.Nk = Nk;
  a.d = d;
  a.scale = scale;
  a.accumulate_dq = accumulate_dq;
  a.stream = static_cast<hipStream_t>(stream);
  return a;
}

int vitattn_bwd(const void* q, const void* k, const void* v, const float* o, const void* dout, const float* lse,
                float* dq, float* dk, float* dv, int B, int H, int N, int d, float scale, void* workspace,
                size_t workspace_bytes, void* stream) {
  return vitattn_bwd_kv(q, k, v, o, dout, lse, dq, dk, dv, B, H, N, N, d, scale, 0, workspace, workspace_bytes,
                        stream);
}

int vitattn_bwd_kv(const void* q, const void* k, const void* v, const float* o, const void* dout, const float* lse,
                   float* dq, float* dk, float* dv, int B, int H, int Nq, int Nk, int d, float scale, int flags,
                   void* workspace, size_t workspace_bytes, void* stream) {
  const vitattn_strides mq = dense(H, Nq, d), mk = dense(H, Nk, d);
  return vitattn_bwd_strided(q, mq, k, mk, v, mk, o, mq, dout, mq, lse, dq, mq, dk, mk, dv, mk, B, H, Nq, Nk, d,
                             scale, flags, workspace, workspace_bytes, stream);
}

int vitattn_bwd_strided(const void* q, vitattn_strides sq, const void* k, vitattn_strides sk, const void* v,
                        vitattn_strides sv, const float* o, vitattn_strides so, const void* dout,
                        vitattn_strides sdo, const float* lse, float* dq, vitattn_strides sdq, float* dk,
                        vitattn_strides sdk, float* dv, vitattn_strides sdv, int B, int H, int Nq, int Nk, int d,
                        float scale, int flags, void* workspace, size_t workspace_bytes, void* stream) {
  try {
    int st = check_sizes_kv(B, H, Nq, Nk, d);
    if (st != VITATTN_OK) return st;
    if (!bwd_items_ok(B, H, Nq, Nk, d)) return VITATTN_E_INVAL;
    if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(o) || !aligned16(dout) || !aligned16(lse) ||
        !aligned16(dq) || !aligned16(dk) || !aligned16(dv))
      return VITATTN_E_INVAL;
    if (!scale_ok(scale)) return VITATTN_E_INVAL;
    if ((flags & ~(VITATTN_BWD_ACCUMULATE_DQ | VITATTN_BWD_STORE_DS)) != 0) return VITATTN_E_INVAL;
    if ((flags & VITATTN_BWD_STORE_DS) && !ds_mode_ok(Nq)) return VITATTN_E_INVAL;
    if (check_map(sq, B, H, Nq, d, 2, false) || check_map(sk, B, H, Nk, d, 2, false) ||
        check_map(sv, B, H, Nk, d, 2, false) || check_map(so, B, H, Nq, d, 4, false) ||
        check_map(sdo, B, H, Nq, d, 2, false) || check_map(sdq, B, H, Nq, d, 4, true) ||
        check_map(sdk, B, H, Nk, d, 4, true) || check_map(sdv, B, H, Nk, d, 4, true))
      return VITATTN_E_INVAL;
    if (workspace == nullptr || (reinterpret_cast<uintptr_t>(workspace) & 15u) != 0 ||
        workspace_bytes < vitattn_bwd_workspace_bytes_kv(B, H, Nq, Nk, d, flags))
      return VITATTN_E_WORKSPACE;
    vitattn::BwdArgs a = bwd_args(q, k, v, o, dout, lse, dq, dk, dv, B, H, Nq, Nk, d, scale,
                                  (flags & VITATTN_BWD_ACCUMULATE_DQ) != 0, workspace, stream);
    if (flags & VITATTN_BWD_STORE_DS)
      a.ds = reinterpret_cast<uint16_t*>(static_cast<char*>(workspace) + vitattn_bwd_workspace_bytes(B, H, Nq, d));
    a.mq = to_map(sq);
    a.mk = to_map(sk);
    a.mv = to_map(sv);
    a.mo = to_map(so);
    a.mg = to_map(sdo);
    a.mdq = to_map(sdq);
    a.mdk = to_map(sdk);
    a.mdv = to_map(sdv);
    return vitattn::launch_bwd(a) == hipSuccess ? VITATTN_OK : VITATTN_E_HIP;
  } catch (...) {
    return VITATTN_E_INTERNAL;
  }
}

int vitattn_merge(const float* o_parts, const float* lse_parts, int n_parts, float* o, float* lse, int B, int H,
                  int N, int d, void* stream) {
  try {
    int st = check_sizes(B, H, N, d);  // d: a multiple of 8 up to 160, as for the attention
    if (st != VITATTN_OK) return st;
    if (!merge_items_ok(B, H, N, d)) return VITATTN_E_INVAL;
    if (n_parts < 1 || n_parts > VITATTN_MERGE_MAX_PARTS) return VITATTN_E_INVAL;
    if (!aligned16(o_parts) || !aligned16(lse_parts) || !aligned16(o) || !aligned16(lse)) return VITATTN_E_INVAL;
    vitattn::MergeArgs a;
    a.o_parts = o_parts;
    a.lse_parts = lse_parts;
    a.o = o;
    a.lse = lse;
    a.P = n_parts;
    a.BH = B * H;
    a.N = N;
    a.d = d;
    a.stream = static_cast<hipStream_t>(stream);
    return vitattn::launch_merge(a) == hipSuccess ? VITATTN_OK : VITATTN_E_HIP;
  } catch (...) {
    return VITATTN_E_INTERNAL;
  }
}

int vitattn_bwd_rowdot(const float* o, const void* dout, const float* lse, int B, int H, int N, int d,
                       void* workspace, size_t workspace_bytes, void* stream) {
  try {
    int st = check_sizes(B, H, N, d);
    if (st != VITATTN_OK) return st;
    if (!bwd_items_ok(B, H, N, N, d)) return VITATTN_E_INVAL;
    if (!aligned16(o) || !aligned16(dout) || !aligned16(lse)) return VITATTN_E_INVAL;
    st = check_workspace(workspace, workspace_bytes, B, H, N, d);
    if (st != VITATTN_OK) return st;
    const vitattn::BwdArgs a = bwd_args(nullptr, nullptr, nullptr, o, dout, lse, nullptr, nullptr, nullptr, B, H, N,
                                        N, d, 1.f, false, workspace, stream);
    return vitattn::launch_bwd_rowdot(a) == hipSuccess ? VITATTN_OK : VITATTN_E_HIP;
  } catch (...) {
    return VITATTN_E_INTERNAL;
  }
}

int vitattn_bwd_dkdv(const void* q, const void* k, const void* v, const void* dout, const float* lse, float* dk,
                     float* dv, int B, int H, int N, int d, float scale, const void* workspace,
                     size_t workspace_bytes, void* stream) {
  try {
    int st = check_sizes(B, H, N, d);
    if (st != VITATTN_OK) return st;
    if (!bwd_items_ok(B, H, N, N, d)) return VITATTN_E_INVAL;
    if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(dout) || !aligned16(lse) || !aligned16(dk) ||
        !aligned16(dv))
      return VITATTN_E_INVAL;
    if (!scale_ok(scale)) return VITATTN_E_INVAL;
    st = check_workspace(workspace, workspace_bytes, B, H, N, d);
    if (st != VITATTN_OK) return st;
    const vitattn::BwdArgs a =
        bwd_args(q, k, v, nullptr, dout, lse, nullptr, dk, dv, B, H, N, N, d, scale, false, workspace, stream);
    return vitattn::launch_bwd_dkdv(a) == hipSuccess ? VITATTN_OK : VITATTN_E_HIP;
  } catch (...) {
    return VITATTN_E_INTERNAL;
  }
}

int vitattn_bwd_dq(const void* q, const void* k, const void* v, const void* dout, const float* lse, float* dq,
                   int B, int H, int N, int d, float scale, const void* workspace, size_t workspace_bytes,
                   void* stream) {
  try {
    int st = check_sizes(B, H, N, d);
    if (st != VITATTN_OK) return st;
    if (!bwd_items_ok(B, H, N, N, d)) return VITATTN_E_INVAL;
    if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(dout) || !aligned16(lse) || !aligned16(dq))
      return VITATTN_E_INVAL;
    if (!scale_ok(scale)) return VITATTN_E_INVAL;
    st = check_workspace(workspace, workspace_bytes, B, H, N, d);
    if (st != VITATTN_OK) return st;
    const vitattn::BwdArgs a =
        bwd_args(q, k, v, nullptr, dout, lse, dq, nullptr, nullptr, B, H, N, N, d, scale, false, workspace, stream);
    return vitattn::launch_bwd_dq(a) == hipSuccess ? VITATTN_OK : VITATTN_E_HIP;
  } catch (...) {
    return VITATTN_E_INTERNAL;
  }
}

static int ulysses(const void* src, void* dst, int B, int Nl, int H, int P, int row_bytes, int mode, void* stream) {
  try {
    if (B < 1 || Nl < 1 || H < 1 || P < 1 || H % P != 0) return VITATTN_E_INVAL;
    if (row_bytes < 16 || row_bytes % 16 != 0) return VITATTN_E_INVAL;
    if (!aligned16(src) || !aligned16(dst) || src == dst) return VITATTN_E_INVAL;
    // grid limits: B indexes grid.y, (token tiles x H) grid.x, Nl*row_bytes/16 a 32-bit thread index
    if (B > 65535 || (long long)Nl * (row_bytes / 16) > 0x7fffffffLL) return VITATTN_E_INVAL;
    if (vitattn::ulysses_blocks(Nl, H, row_bytes) * 256 >= kMaxWorkItems) return VITATTN_E_INVAL;  // 256 per block
    if ((double)B * Nl * H * row_bytes > 9.0e18) return VITATTN_E_INVAL;
    vitattn::UlyssesArgs a;
    a.src = src;
    a.dst = dst;
    a.B = B;
    a.Nl = Nl;
    a.H = H;
    a.P = P;
    a.row_bytes = row_bytes;
    a.mode = mode;
    a.stream = static_cast<hipStream_t>(stream);
    return vitattn::launch_ulysses(a) == hipSuccess ? VITATTN_OK : VITATTN_E_HIP;
  } catch (...) {
    return VITATTN_E_INTERNAL;
  }
}

int vitattn_ulysses_pack(const void* x, void* send, int B, int Nl, int H, int P, int row_bytes, void* stream) {
  return ulysses(x, send, B, Nl, H, P, row_bytes, vitattn::kUlyssesPack, stream);
}

int vitattn_ulysses_unpack(const void* recv, void* y, int B, int Nl, int H, int P, int row_bytes, void* stream) {
  return ulysses(recv, y, B, Nl, H, P, row_bytes, vitattn::kUlyssesUnpack, stream);
}

int vitattn_ulysses_pack_out(const void* y, void* send, int B, int Nl, int H, int P, int row_bytes, void* stream) {
  return ulysses(y, send, B, Nl, H, P, row_bytes, vitattn::kUlyssesPackOut, stream);
}

int vitattn_ulysses_unpack_out(const void* recv, void* x, int B, int Nl, int H, int P, int row_bytes,
                               void* stream) {
  return ulysses(recv, x, B, Nl, H, P, row_bytes, vitattn::kUlyssesUnpackOut, stream);
}

static int check_agg(int M, int H, int C, int d, float scale) {
  if (M < 1 || H < 1 || C < 1) return VITATTN_E_INVAL;
  if (d != 64 && d != 128) return VITATTN_E_UNSUPPORTED;
  if ((long long)M * H > 0x7fffffffLL || (long long)H * d > 0x7fffffffLL) return VITATTN_E_INVAL;
  // launches below 2^32 work-items: 64 per (patch, head) in the forward and
  // backward (patches in groups of four), 64 per dq column in its reduction
  if ((M + 3LL) * H * 64 >= kMaxWorkItems || ((long long)H * d + 15) * 64 >= kMaxWorkItems) return VITATTN_E_INVAL;
  if ((double)M * H * C * d > 4.0e18) return VITATTN_E_INVAL;
  return scale_ok(scale) ? VITATTN_OK : VITATTN_E_INVAL;
}

size_t vitattn_agg_bwd_workspace_bytes(int M, int H, int C, int d) {
  if (check_agg(M, H, C, d, 1.f) != VITATTN_OK) return 0;
  return (size_t)vitattn::agg_partials(M) * H * d * sizeof(float);
}

int vitattn_agg_fwd(const void* q, const void* k, const void* v, float* o, float* lse, int M, int H, int C, int d,
                    float scale, void* stream) {
  try {
    const int st = check_agg(M, H, C, d, scale);
    if (st != VITATTN_OK) return st;
    if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(o) || !aligned16(lse)) return VITATTN_E_INVAL;
    vitattn::AggArgs a = {};
    a.q = static_cast<const uint16_t*>(q);
    a.k = static_cast<const uint16_t*>(k);
    a.v = static_cast<const uint16_t*>(v);
    a.o_out = o;
    a.lse_out = lse;
    a.M = M;
    a.H = H;
    a.C = C;
    a.d = d;
    a.scale = scale;
    a.stream = static_cast<hipStream_t>(stream);
    return vitattn::launch_agg_fwd(a) == hipSuccess ? VITATTN_OK : VITATTN_E_HIP;
  } catch (...) {
    return VITATTN_E_INTERNAL;
  }
}

int vitattn_agg_bwd(const void* q, const void* k, const void* v, const float* o, const void* dout, const float* lse,
                    float* dq, float* dk, float* dv, int M, int H, int C, int d, float scale, void* workspace,
                    size_t workspace_bytes, void* stream) {
  try {
    int st = check_agg(M, H, C, d, scale);
    if (st != VITATTN_OK) return st;
    if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(o) || !aligned16(dout) || !aligned16(lse) ||
        !aligned16(dq) || !aligned16(dk) || !aligned16(dv))
      return VITATTN_E_INVAL;
    if (workspace == nullptr || !aligned16(workspace) ||
        workspace_bytes < vitattn_agg_bwd_workspace_bytes(M, H, C, d))
      return VITATTN_E_WORKSPACE;
    vitattn::AggArgs a = {};
    a.q = static_cast<const uint16_t*>(q);
    a.k = static_cast<const uint16_t*>(k);
    a.v = static_cast<const uint16_t*>(v);
    a.o = o;
    a.dout = static_cast<const uint16_t*>(dout);
    a.lse = lse;
    a.dq = dq;
    a.dk = dk;
    a.dv = dv;
    a.partial = static_cast<float*>(workspace);
    a.M = M;
    a.H = H;
    a.C = C;
    a.d = d;
    a.scale = scale;
    a.stream = static_cast<hipStream_t>(stream);
    return vitattn::launch_agg_bwd(a) == hipSuccess ? VITATTN_OK : VITATTN_E_HIP;
  } catch (...) {
    return VITATTN_E_INTERNAL;
  }
}

}  // extern "C"

// ------------------------------------------------------------ allocation-free backward
//
// The backward pass's only scratch memory is its workspace: the row statistic
// D and LSE*log2(e), one float each per query row. vitattn_bwd_noalloc keeps
// them in this file-scope array instead of a caller's buffer, sized for
// VITATTN_NOALLOC_MAX_ROWS rows (32 MiB; every device the library runs on
// holds its own copy until the process ends). In host code `scratch` names a
// host-side stand-in, not device memory: kernels get the device address that
// hipGetSymbolAddress returns, looked up once per device with that device
// current. Every call on a device shares that device's copy, and the row
// kernel rewrites every row the later kernels read, so nothing is cleared
// between calls; calls that overlap on one device race.
namespace {
// D and LSE*log2(e), each region padded like the workspace (bwd_region_floats)
constexpr size_t kNoAllocScratchFloats = 2 * (((size_t)VITATTN_NOALLOC_MAX_ROWS + 63) / 64 * 64);
static_assert(kNoAllocScratchFloats * sizeof(float) == (32u << 20), "32 MiB of scratch");
constexpr int kMaxDevices = 64;
}  // namespace

static __device__ __align__(256) float scratch[kNoAllocScratchFloats];

// Device address of this device's copy of `scratch` (nullptr on a HIP error).
static void* noalloc_scratch() {
  static std::mutex mu;
  static void* ptrs[kMaxDevices] = {};
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
  std::lock_guard<std::mutex> lock(mu);
  if (ptrs[dev] == nullptr) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess) return nullptr;
    ptrs[dev] = p;
  }
  return ptrs[dev];
}

extern "C" {

int vitattn_bwd_noalloc(const void* q, const void* k, const void* v, const float* o, const void* dout,
                        const float* lse, float* dq, float* dk, float* dv, int B, int H, int N, int d, float scale,
                        void* stream) {
  try {
    int st = check_sizes(B, H, N, d);
    if (st != VITATTN_OK) return st;
    if (!bwd_items_ok(B, H, N, N, d)) return VITATTN_E_INVAL;
    if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(o) || !aligned16(dout) || !aligned16(lse) ||
        !aligned16(dq) || !aligned16(dk) || !aligned16(dv))
      return VITATTN_E_INVAL;
    if (!scale_ok(scale)) return VITATTN_E_INVAL;
    const long long rows = (long long)B * H * N;
    if (rows > VITATTN_NOALLOC_MAX_ROWS) return VITATTN_E_TOO_LARGE;
    void* ws = noalloc_scratch();
    if (ws == nullptr) return VITATTN_E_HIP;
    const vitattn::BwdArgs a =
        bwd_args(q, k, v, o, dout, lse, dq, dk, dv, B, H, N, N, d, scale, false, ws, stream);
    return vitattn::launch_bwd(a) == hipSuccess ? VITATTN_OK : VITATTN_E_HIP;
  } catch (...) {
    return VITATTN_E_INTERNAL;
  }
}

// Stages of the dS-mode backward (dense operands), for timing each kernel.
int vitattn_bwd_dkdv_ds(const void* q, const void* k, const void* v, const void* dout, const float* lse, float* dk,
                        float* dv, int B, int H, int N, int d, float scale, void* workspace, size_t workspace_bytes,
                        void* stream) {
  try {
    int st = check_sizes(B, H, N, d);
    if (st != VITATTN_OK) return st;
    if (!bwd_items_ok(B, H, N, N, d)) return VITATTN_E_INVAL;
    if (!aligned16(q) || !aligned16(k) || !aligned16(v) || !aligned16(dout) || !aligned16(lse) || !aligned16(dk) ||
        !aligned16(dv))
      return VITATTN_E_INVAL;
    if (!scale_ok(scale) || !ds_mode_ok(N)) return VITATTN_E_INVAL;
    if (workspace == nullptr || !aligned16(workspace) ||
        workspace_bytes < vitattn_bwd_workspace_bytes_kv(B, H, N, N, d, VITATTN_BWD_STORE_DS))
      return VITATTN_E_WORKSPACE;
    vitattn::BwdArgs a =
        bwd_args(q, k, v, nullptr, dout, lse, nullptr, dk, dv, B, H, N, N, d, scale, false, workspace, stream);
    a.ds = reinterpret_cast<uint16_t*>(static_cast<char*>(workspace) + vitattn_bwd_workspace_bytes(B, H, N, d));
    return vitattn::launch_bwd_dkdv(a) == hipSuccess ? VITATTN_OK : VITATTN_E_HIP;
  } catch (...) {
    return VITATTN_E_INTERNAL;
  }
}

int vitattn_bwd_dq_from_ds(const void* k, float* dq, int B, int H, int N, int d, float scale, const void* workspace,
                           size_t workspace_bytes, void* stream) {
  try {
    int st = check_sizes(B, H, N, d);
    if (st != VITATTN_OK) return st;
    if (!bwd_items_ok(B, H, N, N, d)) return VITATTN_E_INVAL;
    if (!aligned16(k) || !aligned16(dq)) return VITATTN_E_INVAL;
    if (!scale_ok(scale) || !ds_mode_ok(N)) return VITATTN_E_INVAL;
    if (workspace == nullptr || !aligned16(workspace) ||
        workspace_bytes < vitattn_bwd_workspace_bytes_kv(B, H, N, N, d, VITATTN_BWD_STORE_DS))
      return VITATTN_E_WORKSPACE;
    vitattn::BwdArgs a =
        bwd_args(nullptr, k, nullptr, nullptr, nullptr, nullptr, dq, nullptr, nullptr, B, H, N, N, d, scale, false,
                 workspace, stream);
    a.ds = reinterpret_cast<uint16_t*>(static_cast<char*>(const_cast<void*>(workspace)) +
                                       vitattn_bwd_workspace_bytes(B, H, N, d));
    return vitattn::launch_bwd_dq(a) == hipSuccess ? VITATTN_OK : VITATTN_E_HIP;
  } catch (...) {
    return VITATTN_E_INTERNAL;
  }
}

}  // extern "C"
