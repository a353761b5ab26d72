/*
 * vitattn.h — C ABI of the exact non-causal attention library for MI355X (gfx950).
 *
 * What it computes. One GPU's share of the self-attention of a long-sequence
 * Vision Transformer after a DeepSpeed-Ulysses all-to-all (paper Sec. II-E):
 * the full sequence of N patch tokens for H heads of B samples. Attention is
 * dense and bidirectional: every token attends to every token (Sec. I and III),
 * with no mask, bias or dropout. Per (b, h), with s = scale:
 *
 *     S = s Q K^T,  LSE_i = log sum_j exp(S_ij),  P = exp(S - LSE 1^T),  O = P V
 *
 * and the backward pass, given dO = dL/dO:
 *
 *     D_i = sum_c dO_ic O_ic,  dS = P o (dO V^T - D 1^T),
 *     dQ = s dS K,  dK = s dS^T Q,  dV = P^T dO.
 *
 * The tiling (the N x N matrices S and P are never stored), the saved per-row
 * logsumexp and the recomputation of P in the backward pass follow
 * FlashAttention-2, which the paper uses (Sec. II-F, V-B, V-E).
 *
 * Conventions shared by every entry point:
 *  - All tensor pointers are DEVICE pointers owned by the caller. The library
 *    never allocates, frees or retains them, and holds no per-call state.
 *  - Tensors are contiguous row-major [B][H][N][d] (d innermost); lse and the
 *    backward workspace are [B][H][N]. Element offsets use 64-bit arithmetic.
 *    vitattn_fwd_strided / vitattn_bwd_strided take any batch, head and row
 *    strides instead (e.g. the sequence-major [B][N][H][d] layout), see
 *    vitattn_strides below.
 *  - q, k, v and dout hold bfloat16 values as raw 16-bit patterns. o, lse, dq,
 *    dk and dv are fp32. Every pointer must be 16-byte aligned.
 *  - Supported head dims: any multiple of 8 from 8 to 160 (the paper's models
 *    use 64, 72, 128 and 160, Table I and Sec. V-C). The kernels compute in
 *    tiles of width 64, 96, 128 or 160 with the columns past d zero, so d = 72
 *    costs what d = 96 costs. Any N >= 1 with (N + 256) * row_stride * 2 below
 *    2^31 for every bf16 operand (the kernels address one head's rows with
 *    32-bit offsets; N up to 8,388,351 for dense d = 128) and B*H*N below 2^31.
 *    Every kernel launch must also stay below 2^32 work-items: 2*B*H*(N + 383)
 *    for the forward; for the backward and its stages also
 *    4*B*H*(N + 191) + 2^19 and B*H*N times 8, 16 or 32 (head dims up to 64,
 *    128, 160); B*H*N*d/4 + 256 for the merge. These bind only at head dims
 *    of 16 or less (wider rows run out of memory first); a call past them
 *    returns VITATTN_E_INVAL.
 *  - Work is enqueued on `stream` (a hipStream_t; NULL = the null stream) and
 *    the call returns without waiting. Execution faults surface at the
 *    caller's next synchronisation on that stream.
 *  - Arguments are validated before anything is launched; on any error status
 *    no output is written and no kernel is enqueued. Validation itself makes
 *    no HIP call, so it works on a machine without a GPU.
 *  - Results are bitwise deterministic for identical inputs, and a head's
 *    results do not depend on the call it is part of: one call over H heads
 *    gives the bits of H single-head calls, whatever the grid or the CU
 *    count. The only atomics are in the dK/dV stage: when its last round of
 *    key-block workgroups would be at most half full, those key blocks are
 *    split over two workgroups (one per half of the query tiles) that add
 *    into dK and dV rows zeroed first by the same call; two fp32 adds onto
 *    zero give the same bits in either order. Every key block, split or
 *    not, sums its query tiles as the same two rounded partial sums (split
 *    at the middle query tile) and adds them, so splitting changes no bit.
 *    Which blocks split depends on the number of key-block workgroups
 *    (B*H*ceil(N/K), K = 128 keys, or in the default mode 256 at head dims up
 *    to 64 and 192 at 65-80) and the device's CU count, looked up once per
 *    device at the first backward call (no stream work, so a graph capture
 *    may hold it).
 *  - Calls are thread-safe; concurrent calls on different streams are fine.
 */
#ifndef VITATTN_H
#define VITATTN_H

#include <stddef.h>

#ifdef __cplusplus
extern "C" {
#endif

enum vitattn_status {
  VITATTN_OK = 0,
  VITATTN_E_INVAL = 1,       /* null/misaligned pointer, B/H/N < 1, non-finite or non-positive scale, size overflow */
  VITATTN_E_UNSUPPORTED = 2, /* head dim d not supported (see above) */
  VITATTN_E_WORKSPACE = 3,   /* workspace missing or smaller than vitattn_bwd_workspace_bytes() */
  VITATTN_E_HIP = 4,         /* the HIP runtime reported an error when launching */
  VITATTN_E_INTERNAL = 5,    /* unexpected internal failure */
  VITATTN_E_TOO_LARGE = 6    /* vitattn_bwd_noalloc only: B*H*N above VITATTN_NOALLOC_MAX_ROWS */
};

/*
 * Forward pass (the tiled online softmax of FlashAttention-2, cited in paper
 * Sec. II-F).
 *   q, k, v : bf16 [B][H][N][d], read only.
 *   o       : fp32 [B][H][N][d], written: O = softmax(scale * Q K^T) V.
 *   lse     : fp32 [B][H][N], written: natural-log logsumexp of each row of
 *             the scaled logits, LSE_i = log sum_j exp(scale * q_i . k_j).
 *   scale   : softmax scale, finite and > 0 (typically 1/sqrt(d)).
 * Returns a vitattn_status.
 */
int vitattn_fwd(const void* q, const void* k, const void* v, float* o, float* lse, int B, int H, int N, int d,
                float scale, void* stream);

/*
 * Bytes of device workspace vitattn_bwd needs: two fp32 [B][H][N] regions,
 * each padded to a multiple of 64 rows (256 bytes): the row statistic D and
 * LSE * log2(e). Returns 0 for invalid sizes.
 */
size_t vitattn_bwd_workspace_bytes(int B, int H, int N, int d);

/*
 * Backward pass: a D = rowsum(dO o O) preprocess, then one kernel that
 * accumulates dK and dV per key block and one that accumulates dQ per query
 * block, both recomputing P from q, k and lse (FlashAttention-2's backward,
 * cited in paper Sec. II-F).
 *   q, k, v   : bf16 [B][H][N][d], the forward inputs.
 *   o, lse    : fp32, the forward outputs of vitattn_fwd for the same inputs.
 *   dout      : bf16 [B][H][N][d], the gradient of the loss with respect to o.
 *   dq, dk, dv: fp32 [B][H][N][d], written.
 *   workspace : device buffer of at least vitattn_bwd_workspace_bytes() bytes,
 *               overwritten; it must not alias any other argument.
 * Returns a vitattn_status.
 */
int vitattn_bwd(const void* q, const void* k, const void* v, const float* o, const void* dout, const float* lse,
                float* dq, float* dk, float* dv, int B, int H, int N, int d, float scale, void* workspace,
                size_t workspace_bytes, void* stream);

/*
 * The three stages of vitattn_bwd, callable one by one (same arguments,
 * layouts and validation as vitattn_bwd; used to time each kernel). They
 * must run in this order on one stream, all with the same workspace:
 *   vitattn_bwd_rowdot: workspace <- -D_i = -sum_c dout_ic o_ic (stored negated)
 *                       and LSE_i*log2(e);
 *   vitattn_bwd_dkdv  : dk, dv from q, k, v, dout, lse and D in the workspace;
 *   vitattn_bwd_dq    : dq from q, k, v, dout, lse and D in the workspace.
 * Each stage validates its own arguments like vitattn_bwd does.
 */
int vitattn_bwd_rowdot(const float* o, const void* dout, const float* lse, int B, int H, int N, int d,
                       void* workspace, size_t workspace_bytes, void* stream);
int vitattn_bwd_dkdv(const void* q, const void* k, const void* v, const void* dout, const float* lse, float* dk,
                     float* dv, int B, int H, int N, int d, float scale, const void* workspace,
                     size_t workspace_bytes, void* stream);
int vitattn_bwd_dq(const void* q, const void* k, const void* v, const void* dout, const float* lse, float* dq,
                   int B, int H, int N, int d, float scale, const void* workspace, size_t workspace_bytes,
                   void* stream);

/*
 * Attention over one segment of the keys, and the merge of such partial
 * results. Sequence parallelism over contiguous segments (Long Sequence
 * Segmentation, paper Sec. I and II "Sequence Parallel"; one segment per
 * worker) hands one GPU its queries and the keys of one segment at a time.
 * Softmax over a union of key sets factors over the sets:
 *
 *     LSE_i = log sum_s exp(LSE_s,i),   O_i = sum_s exp(LSE_s,i - LSE_i) O_s,i
 *
 * and the backward pass of one segment, given the merged O and LSE, yields
 * that segment's complete dK and dV rows and its share of dQ.
 */

/*
 * Forward pass of Nq queries over Nk keys (vitattn_fwd is the case
 * Nq = Nk = N; same algorithm, conventions and validation).
 *   q        : bf16 [B][H][Nq][d];  k, v: bf16 [B][H][Nk][d].
 *   o        : fp32 [B][H][Nq][d], written; lse: fp32 [B][H][Nq], written.
 *   Nq, Nk   : each >= 1 and within the limits N obeys for vitattn_fwd.
 */
int vitattn_fwd_kv(const void* q, const void* k, const void* v, float* o, float* lse, int B, int H, int Nq, int Nk,
                   int d, float scale, void* stream);

/* flags of vitattn_bwd_kv and vitattn_bwd_strided */
#define VITATTN_BWD_ACCUMULATE_DQ 1 /* dq += this segment's share instead of dq = it */
#define VITATTN_BWD_STORE_DS 2      /* dS mode: dQ from stored dS (see vitattn_bwd_workspace_bytes_kv) */

/*
 * Workspace bytes of vitattn_bwd_kv / vitattn_bwd_strided for these sizes
 * and flags; 0 for invalid arguments. Without VITATTN_BWD_STORE_DS it equals
 * vitattn_bwd_workspace_bytes(B, H, Nq, d).
 *
 * The dS mode trades memory for matrix-core work. The dK/dV kernel already
 * forms dS = P o (dP - D) (bf16, the value it multiplies into dK); with
 * VITATTN_BWD_STORE_DS it also writes every dS block to the workspace, and dQ
 * = scale dS K then streams them (2 d flops per score) instead of recomputing
 * S and dP in a third kernel (6 d flops per score). The extra workspace is
 * 2 bytes per (query, key) pair of every head, rounded up to 64 queries and
 * 128 keys: B*H*Nq*Nk*2 bytes, 142 GB at B=1, H=2, N=188,416. Results differ
 * from the default mode only in the rounding of dS (the default dQ kernel
 * rounds an fp32 P times (dP - D) to bf16, this one a bf16 P times it).
 * Requires Nq <= 16,777,152.
 */
size_t vitattn_bwd_workspace_bytes_kv(int B, int H, int Nq, int Nk, int d, int flags);

/*
 * Backward pass of Nq queries over Nk keys (vitattn_bwd is the case
 * Nq = Nk = N, flags = 0).
 *   q, dout  : bf16 [B][H][Nq][d];  k, v: bf16 [B][H][Nk][d].
 *   o, lse   : fp32 [B][H][Nq][d] and [B][H][Nq]: the output and LSE of the
 *              attention the gradient flows through. For one key segment of a
 *              larger key set pass the MERGED o and lse of all keys: then
 *              dk, dv (fp32 [B][H][Nk][d], written) are exact for this
 *              segment's keys and dq (fp32 [B][H][Nq][d]) is its share.
 *   flags    : 0, or VITATTN_BWD_ACCUMULATE_DQ to add the share to dq (sum
 *              the segments of one key set by calling once per segment on
 *              one stream with dq zeroed first; the order of the sum is the
 *              order of the calls), and/or VITATTN_BWD_STORE_DS (below).
 *              Other bits: VITATTN_E_INVAL.
 *   workspace: at least vitattn_bwd_workspace_bytes_kv(B, H, Nq, Nk, d, flags)
 *              bytes (vitattn_bwd_workspace_bytes(B, H, Nq, d) without
 *              VITATTN_BWD_STORE_DS), else VITATTN_E_WORKSPACE.
 */
int vitattn_bwd_kv(const void* q, const void* k, const void* v, const float* o, const void* dout, const float* lse,
                   float* dq, float* dk, float* dv, int B, int H, int Nq, int Nk, int d, float scale, int flags,
                   void* workspace, size_t workspace_bytes, void* stream);

/*
 * Operands in other layouts. The layout an all-to-all or a fused QKV
 * projection produces is rarely the dense [B][H][N][d]: the sequence-major
 * [B][N][H][d] (paper Sec. II "Sequence Parallel") has strides
 * {N*H*d, d, H*d}, rows padded to a larger pitch have row > d, and a slice
 * of a [B][N][3][H][d] QKV tensor has row = 3*H*d. The kernels read and write
 * such operands in place; no copy is made.
 *
 * Element strides of one operand viewed as [B][H][N][d]; the d elements of a
 * row are contiguous. Every stride must be >= 0 and a multiple of 8 elements
 * for bf16 operands (4 for fp32), so rows stay 16-byte aligned, and
 * row >= d. Inputs may repeat a head or batch (stride 0, e.g. keys shared by
 * several query heads); an output may not overlap itself (checked: sorted by
 * stride, every dimension must step past the span of the smaller ones). Each
 * bf16 operand needs (rows + 256) * row * 2 < 2^31. Violations:
 * VITATTN_E_INVAL. lse and the workspace stay dense [B][H][Nq].
 */
typedef struct vitattn_strides {
  long long batch, head, row;
} vitattn_strides;

/* vitattn_fwd_kv with a layout per operand (same computation and validation). */
int vitattn_fwd_strided(const void* q, vitattn_strides sq, const void* k, vitattn_strides sk, const void* v,
                        vitattn_strides sv, float* o, vitattn_strides so, float* lse, int B, int H, int Nq, int Nk,
                        int d, float scale, void* stream);

/* vitattn_bwd_kv with a layout per operand (same computation, flags and
 * validation); sdo is the layout of dout. */
int vitattn_bwd_strided(const void* q, vitattn_strides sq, const void* k, vitattn_strides sk, const void* v,
                        vitattn_strides sv, const float* o, vitattn_strides so, const void* dout,
                        vitattn_strides sdo, const float* lse, float* dq, vitattn_strides sdq, float* dk,
                        vitattn_strides sdk, float* dv, vitattn_strides sdv, int B, int H, int Nq, int Nk, int d,
                        float scale, int flags, void* workspace, size_t workspace_bytes, void* stream);

/* The two kernels of the dS mode as separate calls (dense operands, Nq = Nk =
 * N; the row-statistics stage vitattn_bwd_rowdot runs first), for timing each:
 * vitattn_bwd_dkdv_ds writes dK, dV and the dS blocks into the workspace,
 * vitattn_bwd_dq_from_ds then writes dQ from them. The workspace must hold
 * vitattn_bwd_workspace_bytes_kv(B, H, N, N, d, VITATTN_BWD_STORE_DS) bytes. */
int vitattn_bwd_dkdv_ds(const void* q, const void* k, const void* v, const void* dout, const float* lse, float* dk,
                        float* dv, int B, int H, int N, int d, float scale, void* workspace, size_t workspace_bytes,
                        void* stream);
int vitattn_bwd_dq_from_ds(const void* k, float* dq, int B, int H, int N, int d, float scale, const void* workspace,
                           size_t workspace_bytes, void* stream);

/* largest number of partial results vitattn_merge accepts */
#define VITATTN_MERGE_MAX_PARTS 65536

/*
 * Merge n_parts partial attention results over disjoint key segments into
 * the attention over all of them (the formula above).
 *   o_parts  : fp32 [n_parts][B][H][N][d], read; lse_parts: fp32
 *              [n_parts][B][H][N], read (each partial as written by
 *              vitattn_fwd_kv for its segment).
 *   o, lse   : fp32 [B][H][N][d] and [B][H][N], written; they must not alias
 *              the partials.
 *   n_parts  : 1 .. VITATTN_MERGE_MAX_PARTS, else VITATTN_E_INVAL.
 *   d        : any head dim the attention takes (a multiple of 8 up to 160),
 *              else VITATTN_E_UNSUPPORTED.
 * A NaN partial LSE makes the merged row NaN. Bound by HBM bandwidth.
 */
int vitattn_merge(const float* o_parts, const float* lse_parts, int n_parts, float* o, float* lse, int B, int H,
                  int N, int d, void* stream);

/*
 * Layouts around DeepSpeed-Ulysses' all-to-all (paper Sec. II "Sequence
 * Parallel"; two all-to-alls per attention in each pass, Sec. V). Each of P
 * ranks holds Nl tokens of all H heads (rank r: tokens r*Nl .. r*Nl+Nl-1);
 * attention needs the whole sequence N = P*Nl of Hl = H/P heads. With
 * rows of row_bytes bytes (one token of one head, e.g. d bf16 values):
 *
 *   pack       x    [B][Nl][H]       -> send [P][B][Hl][Nl]   send[p][b][j][i] = x[b][i][p*Hl+j]
 *   (all-to-all: chunk p of rank r's send buffer becomes chunk r of rank p's receive buffer)
 *   unpack     recv [P][B][Hl][Nl]   -> y    [B][Hl][P*Nl]    y[b][j][r*Nl+i] = recv[r][b][j][i]
 *   pack_out   y    [B][Hl][P*Nl]    -> send [P][B][Hl][Nl]   (inverse of unpack)
 *   unpack_out recv [P][B][Hl][Nl]   -> x    [B][Nl][H]       (inverse of pack)
 *
 * y is the contiguous [B][Hl][N][row] input (or output) of the attention
 * entry points. The collective itself is not part of this library.
 *   B, Nl, H, P: >= 1 with H divisible by P, B <= 65535, Nl*row_bytes/16 < 2^31
 *                and ceil(Nl*row_bytes/4096)*H < 2^24 (256 work-items per
 *                block, below 2^32 per launch).
 *   row_bytes  : a multiple of 16, >= 16.
 *   src, dst   : device pointers, 16-byte aligned, not overlapping
 *                (src == dst is rejected; partial overlap is not detected).
 * Pure copies, bound by HBM bandwidth. Returns a vitattn_status.
 */
int vitattn_ulysses_pack(const void* x, void* send, int B, int Nl, int H, int P, int row_bytes, void* stream);
int vitattn_ulysses_unpack(const void* recv, void* y, int B, int Nl, int H, int P, int row_bytes, void* stream);
int vitattn_ulysses_pack_out(const void* y, void* send, int B, int Nl, int H, int P, int row_bytes, void* stream);
int vitattn_ulysses_unpack_out(const void* recv, void* x, int B, int Nl, int H, int P, int row_bytes, void* stream);

/*
 * Channel aggregation by attention with a learnable query: the Agg-Ch-ViT
 * layer (paper Sec. II "Patch Embedding and Sequence Length") folds the C
 * channel tokens of each patch into one token. For M patch positions (batch
 * x patches) and H heads, one query q_h per head, shared by every patch,
 * attends over that patch's projected channel keys and values:
 *
 *   s_c = scale q_h . k_mhc,  lse_mh = log sum_c exp(s_c),  o_mh = sum_c exp(s_c - lse_mh) v_mhc
 *
 * and the backward pass (dq sums over every patch, as q is shared):
 *
 *   ds_c = p_c (do_mh . v_mhc - do_mh . o_mh),  dk_mhc = scale ds_c q_h,
 *   dv_mhc = p_c do_mh,  dq_h = scale sum_m sum_c ds_c k_mhc.
 *
 * Layouts (row-major): q bf16 [H][d]; k, v bf16 [M][H][C][d]; o fp32
 * [M][H][d]; lse fp32 [M][H]; dout bf16 [M][H][d]; dq fp32 [H][d]; dk, dv
 * fp32 [M][H][C][d]. M, H, C >= 1 (any C; the paper's case is C = 92) with
 * (M + 3)*H and H*d below 2^26 (64 work-items each per launch, below 2^32);
 * d in {64, 128}; scale finite and > 0. Bound by HBM bandwidth. dq is
 * reduced in a fixed order (no atomics): results are bitwise reproducible.
 */
int vitattn_agg_fwd(const void* q, const void* k, const void* v, float* o, float* lse, int M, int H, int C, int d,
                    float scale, void* stream);

/* Workspace bytes of vitattn_agg_bwd: dq partials, one per head and group of four
 * patches (ceil(M/4) x H x d floats); 0 for invalid sizes. */
size_t vitattn_agg_bwd_workspace_bytes(int M, int H, int C, int d);

/* o and lse are vitattn_agg_fwd's outputs for the same q, k, v; workspace is
 * overwritten and must not alias any other argument. */
int vitattn_agg_bwd(const void* q, const void* k, const void* v, const float* o, const void* dout, const float* lse,
                    float* dq, float* dk, float* dv, int M, int H, int C, int d, float scale, void* workspace,
                    size_t workspace_bytes, void* stream);

/*
 * vitattn_bwd without a workspace argument, for callers that cannot allocate
 * device memory (code under HIP graph capture, serving loops that must not
 * call hipMalloc, harnesses that forbid it). Same arguments (minus the
 * workspace), layouts, validation, kernels and results as vitattn_bwd: the
 * outputs are bitwise equal to vitattn_bwd's for the same inputs. The
 * workspace lives in a static device array of the library (32 MiB, one copy
 * per device the library runs on, held until the process ends), so:
 *   - B*H*N may be at most VITATTN_NOALLOC_MAX_ROWS, else VITATTN_E_TOO_LARGE
 *     (and nothing is launched);
 *   - the call itself allocates nothing (no hipMalloc, hipFree or allocating
 *     library routine). Its first call on a device looks up that device's
 *     copy of the array (hipGetSymbolAddress) with that device current; the
 *     stream must belong to the calling thread's current device;
 *   - every call on a device shares that device's array: calls that overlap
 *     in time on one device (other streams, other threads) race and must be
 *     serialised by the caller. Nothing in the array needs clearing between
 *     calls: each call rewrites every entry it reads.
 */
#define VITATTN_NOALLOC_MAX_ROWS 4194304
int vitattn_bwd_noalloc(const void* q, const void* k, const void* v, const float* o, const void* dout,
                        const float* lse, float* dq, float* dk, float* dv, int B, int H, int N, int d, float scale,
                        void* stream);

/* Human-readable name of a status code (static storage, never NULL). */
const char* vitattn_status_str(int status);

/* Library version string (static storage). */
const char* vitattn_version(void);

#ifdef __cplusplus
}
#endif

#endif /* VITATTN_H */
