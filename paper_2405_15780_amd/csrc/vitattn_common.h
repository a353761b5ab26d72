// Device helpers shared by the forward and backward attention kernels (gfx950).
//
// Matrix-core conventions (v_mfma_f32_32x32x16_bf16, wave64):
//   A operand (32 x 16) and B operand (16 x 32) have the same lane layout:
//   lane l holds the 8 contraction elements (l/32)*8 .. (l/32)*8+7 of row
//   (A) or column (B) l%32. The 32 x 32 fp32 accumulator gives lane l the
//   column l%32 and, in register r, the row 8*(r/4) + 4*(l/32) + r%4.
//
// An accumulator whose rows are the next product's contraction index (the
// probabilities P^T, keys x queries, feeding P V) is reused as that
// product's operand without moving data between lanes: registers 8*ks ..
// 8*ks+7 form the operand of contraction step ks, whose slot t of half h
// = l/32 holds row 16*ks + 8*(t/4) + 4*h + t%4. The other operand is then
// gathered with ds_read_b64_tr_b16 from a row-major LDS tile in that same
// row order (frag_tr below), so no tile is ever transposed in memory.
//
// LDS tiles are row-major [rows][D] bf16 with the 16-byte chunks of row r
// XOR-swizzled by swz(r), so that both the row-fragment reads (32 rows x one
// chunk) and the transposing reads (8 rows x 4 chunks) touch every bank
// equally often. The tile width D is 64, 96, 128 or 160; a head dim d below
// D occupies the first d columns and the rest of each row holds zeros.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

namespace vitattn {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

__device__ __forceinline__ f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ f32x16 zero16() {
  f32x16 z;
#pragma unroll
  for (int i = 0; i < 16; ++i) z[i] = 0.f;
  return z;
}

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 u) { return __builtin_bit_cast(bf16x8, u); }

// Swizzled byte offset of 16-byte chunk c of row r in a [rows][D] bf16 tile.
// D = 128 and 64: 16 consecutive rows of one chunk cover all 64 banks. D = 96
// and 160 (rows of 192 and 320 bytes): four consecutive rows already start in
// four different 64-byte bank groups, so the swizzle permutes chunks only
// within their aligned group of four (never past the end of the row) and
// varies with rows 4 apart.
template <int D>
__device__ __forceinline__ int swz(int r) {
  static_assert(D == 64 || D == 96 || D == 128 || D == 160, "tile width");
  if constexpr (D == 128) return ((r & 3) << 2) | ((r >> 2) & 3);
  else if constexpr (D == 64) return (((r >> 1) & 1) << 2) | ((r >> 2) & 3);
  else return (r >> 2) & 3;
}
template <int D>
__device__ __forceinline__ int tile_off(int r, int c) {
  return r * (2 * D) + 16 * (c ^ swz<D>(r));
}

// Row fragment: lane l gets T[r0 + l%32][16*kk + 8*(l/32) .. +7] (an A or B
// operand whose contraction runs along d). `roff` is the lane's precomputed
// tile_off for chunk 2*kk + l/32 of its row, see RowFrag.
__device__ __forceinline__ bf16x8 lds_frag_row(const char* lds, int off) {
  return as_bf16x8(*reinterpret_cast<const uint4*>(lds + off));
}

// Tile widths whose swizzle permutes chunks within aligned groups of four:
// moving a fragment by one group (64 bytes) is then a plain constant offset.
template <int D>
constexpr bool kGrouped = (D == 96 || D == 160);

// Per-lane offsets of the row fragments of rows r0 + l%32 (r0 a multiple of
// 32, added by the caller as r0 * 2D), for every kk = 0 .. D/16 - 1. For the
// grouped widths chunk 2*kk + h sits in group kk/2 at position 2*(kk%2) + h,
// so two registers cover every kk.
template <int D>
struct RowFrag {
  int off_[kGrouped<D> ? 2 : D / 16];
  __device__ __forceinline__ void init(int lane) {
    const int row = lane & 31, h = lane >> 5;
#pragma unroll
    for (int kk = 0; kk < (kGrouped<D> ? 2 : D / 16); ++kk) off_[kk] = tile_off<D>(row, 2 * kk + h);
  }
  __device__ __forceinline__ int at(int kk) const {
    if constexpr (kGrouped<D>) return off_[kk & 1] + 64 * (kk >> 1);
    else return off_[kk];
  }
};

// Transposed fragment: operand whose contraction runs along rows. For
// contraction step base row k0 (a multiple of 16) and column block c0 (a
// multiple of 32), lane l gets T[k0 + 8*(t/4) + 4*(l/32) + t%4][c0 + l%32]
// in slot t = 0..7 — the row order of an accumulator reused as an operand.
// Built from two ds_read_b64_tr_b16: within each 16-lane group, lane i of the
// result takes element i%4 of the 8 bytes addressed by lane 4e + i/4 of the
// group, for e = 0..3. A column block is one chunk group, so for the grouped
// widths block cb is block 0 plus 64*cb bytes.
template <int D>
struct TrFrag {
  static constexpr int NCB = kGrouped<D> ? 1 : D / 32;
  int off[2][NCB];  // [read][column block]
  __device__ __forceinline__ void init(int lane) {
    const int g = lane >> 4, j = lane & 15;
#pragma unroll
    for (int rd = 0; rd < 2; ++rd) {
      const int row = 8 * rd + 4 * (g >> 1) + (j >> 2);
#pragma unroll
      for (int cb = 0; cb < NCB; ++cb) {
        const int col = 32 * cb + 16 * (g & 1) + 4 * (j & 3);
        off[rd][cb] = row * (2 * D) + 16 * ((col >> 3) ^ swz<D>(row)) + 2 * (col & 7);
      }
    }
  }
  // k0: contraction base row (multiple of 16); the row part of the swizzle
  // depends only on the low 4 row bits, so k0 enters as a plain offset.
  __device__ __forceinline__ bf16x8 load(const char* lds, int k0, int cb) const {
    const int o0 = kGrouped<D> ? off[0][0] + 64 * cb : off[0][cb];
    const int o1 = kGrouped<D> ? off[1][0] + 64 * cb : off[1][cb];
    const char* p0 = lds + k0 * (2 * D) + o0;
    const char* p1 = lds + k0 * (2 * D) + o1;
    bf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(p0));
    bf16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(p1));
    bf16x8 r;
    r[0] = lo[0]; r[1] = lo[1]; r[2] = lo[2]; r[3] = lo[3];
    r[4] = hi[0]; r[5] = hi[1]; r[6] = hi[2]; r[7] = hi[3];
    return r;
  }
};

// Accumulator registers 8*ks .. 8*ks+7 -> bf16 operand (round to nearest even).
__device__ __forceinline__ bf16x8 acc_to_operand(const f32x16& a, int ks) {
  bf16x8 r;
#pragma unroll
  for (int t = 0; t < 8; ++t) r[t] = (__bf16)a[8 * ks + t];
  return r;
}

// Row of accumulator register r for lane half h.
__device__ __forceinline__ int acc_row(int r, int h) { return 8 * (r >> 2) + 4 * h + (r & 3); }

// Work-item remap so that consecutive work items land on the same XCD
// (workgroups are dealt round-robin over the 8 XCDs, each with its own L2).
__device__ __forceinline__ int xcd_remap(int bid, int total) {
  constexpr int kXcd = 8;
  const int q = total / kXcd, rem = total % kXcd;
  const int x = bid % kXcd, j = bid / kXcd;
  return x * q + (x < rem ? x : rem) + j;
}

// Value of lane l^32 combined with lane l's own: v_permlane32_swap on (v, v)
// yields v[l%32] and v[32 + l%32] in every lane.
__device__ __forceinline__ float max_halves(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float sum_halves(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ float xor32(float v) { return __shfl_xor(v, 32, 64); }

// ------------------------------------------------------------ buffer loads
// A raw buffer resource over `bytes` bytes from `base`: loads at offsets at
// or past `bytes` return zeros without touching memory, which is how tile
// loads handle the ragged end of a sequence without branches.
typedef __amdgpu_buffer_rsrc_t rsrc_t;
typedef __attribute__((address_space(3))) void lds_void_t;

__device__ __forceinline__ rsrc_t make_rsrc(const void* base, unsigned bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}
__device__ __forceinline__ uint4 buffer_load16(rsrc_t r, int byte_off) {
  return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, byte_off, 0, 0));
}

// Byte offset that lies past every buffer the kernels build (their sizes stay
// below 2^31), so a load from it returns zeros: used for the columns of a
// tile beyond the head dim.
constexpr unsigned kOobOffset = 0x80000000u;

// Byte offset of 16-byte chunk `chunk` of row `row` of a bf16 matrix whose
// rows are ld_bytes apart and hold chr real chunks; chunks past the head dim
// point past the buffer and read as zeros.
__device__ __forceinline__ int chunk_offset(int row, int chunk, int ld_bytes, int chr) {
  return chunk < chr ? row * ld_bytes + 16 * chunk : (int)kOobOffset;
}

// Direct global -> LDS copy of an R x D bf16 tile (rows row0 .. row0+R-1 of
// a matrix behind `r` whose rows are ld_bytes apart and hold chr real 16-byte
// chunks) into the swizzled layout of tile_off. One wave instruction fills
// 1 KB of consecutive LDS (16 bytes per lane), so each lane fetches the chunk
// whose swizzled home is its LDS slot. Rows past the end and chunks past the
// head dim read as zeros. The NW waves of the group split the instructions;
// every wave issues the same number per tile (PER_WAVE), so that one vmcnt
// bound fits all of them: when the instruction count is not a multiple of NW
// the surplus slots repeat other waves' instructions (the same bytes into the
// same LDS slot), and with fewer instructions than waves the waves without
// one issue nothing.
template <int D, int R, int NW>
struct TileDma {
  static constexpr int CH = D / 8;
  static_assert(R * CH % 64 == 0, "a tile is a whole number of 1 KB wave instructions");
  static constexpr int INSTR = R * CH / 64;  // wave instructions per tile
  static constexpr bool ALL_ACTIVE = INSTR >= NW;  // every wave has a share
  static constexpr bool BLOCKED = INSTR % NW == 0 || !ALL_ACTIVE;  // contiguous instructions per wave
  static constexpr int PER_WAVE = ALL_ACTIVE ? (INSTR + NW - 1) / NW : 1;
  unsigned voff[PER_WAVE];  // byte offset of this lane's chunk relative to row0
  int lds_off[BLOCKED ? 1 : PER_WAVE];  // LDS byte offset of this wave's (first) instruction
  bool active;              // false for waves left without work on small tiles

  __device__ __forceinline__ static int instr(int wave, int i) {
    if constexpr (BLOCKED) return (wave * PER_WAVE + i) % INSTR;
    else return (wave + NW * i) % INSTR;
  }
  __device__ __forceinline__ void init(int wave, int lane, int ld_bytes, int chr) {
#pragma unroll
    for (int i = 0; i < PER_WAVE; ++i) {
      const int gi = instr(wave, i);
      const int pos = gi * 64 + lane;  // 16-byte slot in the tile
      const int row = pos / CH, pc = (pos % CH) ^ swz<D>(row);
      voff[i] = (unsigned)chunk_offset(row, pc, ld_bytes, chr);
      if constexpr (!BLOCKED) lds_off[i] = gi * 1024;
    }
    if constexpr (BLOCKED) lds_off[0] = instr(wave, 0) * 1024;
    active = wave * PER_WAVE < INSTR;
  }
  __device__ __forceinline__ char* lds_slot(char* lds_tile, int i) const {
    if constexpr (BLOCKED) return lds_tile + lds_off[0] + i * 1024;
    else return lds_tile + lds_off[i];
  }
  // Instruction i (< PER_WAVE) of this wave's share of the tile; row0 *
  // ld_bytes stays below 2^31, so adding an out-of-range chunk offset cannot
  // wrap around into the buffer.
  __device__ __forceinline__ void issue_one(rsrc_t r, int row0, int ld_bytes, char* lds_tile, int i) const {
    if (!ALL_ACTIVE && !active) return;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void_t*)lds_slot(lds_tile, i), 16,
                                             (int)((unsigned)(row0 * ld_bytes) + voff[i]), 0, 0, 0);
  }
  __device__ __forceinline__ void issue(rsrc_t r, int row0, int ld_bytes, char* lds_tile) const {
#pragma unroll
    for (int i = 0; i < PER_WAVE; ++i) issue_one(r, row0, ld_bytes, lds_tile, i);
  }
};

// Debug builds only (-DVITATTN_DEBUG_LDS_POISON): a kernel first fills its
// LDS buffers with all-ones bytes (NaN as bf16 and as fp32), so that any read
// of LDS that nothing wrote turns its outputs into NaN. Without the define
// this emits no code and no barrier.
template <typename... A>
__device__ __forceinline__ void debug_poison_lds(A&... bufs) {
#ifdef VITATTN_DEBUG_LDS_POISON
  auto fill = [](void* p, unsigned bytes) {
    uint32_t* w = static_cast<uint32_t*>(p);
    for (unsigned i = threadIdx.x; i < bytes / 4; i += blockDim.x) w[i] = 0xffffffffu;
  };
  (fill(static_cast<void*>(&bufs), (unsigned)sizeof(bufs)), ...);
  __syncthreads();
#else
  ((void)bufs, ...);
#endif
}

__device__ __forceinline__ void wait_vmem() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }
// Wait until at most CNT of this wave's vector memory loads are in flight
// (loads complete in issue order for this count).
template <int CNT>
__device__ __forceinline__ void wait_vmem_leave() {
  static_assert(CNT >= 0 && CNT < 64, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(CNT) : "memory");
}

// Workgroup barrier for LDS ring pipelines. The caller first waits for its
// own LDS DMA requests that other waves will read (wait_vmem_leave); this
// waits for the wave's own LDS reads and writes, then barriers. Unlike
// __syncthreads() it does not wait for every outstanding vector-memory
// access, so DMA requests for later tiles stay in flight across it; the
// empty asm statements keep the compiler from moving memory accesses across.
__device__ __forceinline__ void barrier_lds() {
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}

// Full scheduling fence: nothing moves across it. Used to pin an explicit
// software pipeline (each step: one matrix-core op, the LDS read of an
// operand needed a few steps later, a slice of unrelated vector work);
// left alone, the scheduler sinks every LDS read next to its consumer and
// the wave then waits out the LDS latency before every op.
__device__ __forceinline__ void sched_fence() { __builtin_amdgcn_sched_barrier(0); }
// Force a value to be computed before this point (IR passes otherwise sink
// pure arithmetic such as exp2 past the fences, towards its first use).
__device__ __forceinline__ void pin(float& x) { asm volatile("" : "+v"(x)); }

// f(integral_constant<int, I>) for I = B .. E-1, each call inlined with I a
// compile-time constant (a plain unrolled loop leaves the index to the
// unroller, and large bodies then fall back to run-time indexing).
template <int B, int E, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (B < E) {
    f(std::integral_constant<int, B>{});
    static_for<B + 1, E>(f);
  }
}

}  // namespace vitattn
