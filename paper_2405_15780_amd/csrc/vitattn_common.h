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
// LDS tiles are row-major [rows][d] bf16 with the 16-byte chunks of row r
// XOR-swizzled by swz(r), so that both the row-fragment reads (32 rows x one
// chunk) and the transposing reads (8 rows x 4 chunks) touch every bank
// equally often.
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
template <int D>
__device__ __forceinline__ int swz(int r) {
  if constexpr (D == 128) return ((r & 3) << 2) | ((r >> 2) & 3);
  else return (((r >> 1) & 1) << 2) | ((r >> 2) & 3);
}
template <int D>
__device__ __forceinline__ int tile_off(int r, int c) {
  return r * (2 * D) + 16 * (c ^ swz<D>(r));
}

// Global -> registers: a tile of R rows x D bf16 starting at row0 of a
// contiguous [N][D] matrix; rows at or past N read as zeros.
template <int D, int R, int NT>
struct TileLoader {
  static constexpr int CH = D / 8;                 // 16-byte chunks per row
  static constexpr int PER_THREAD = R * CH / NT;   // chunks per thread
  static_assert(R * CH % NT == 0, "tile must divide evenly among threads");
  uint4 r[PER_THREAD];

  __device__ __forceinline__ void load(const uint16_t* __restrict__ base, int row0, int N, int tid) {
#pragma unroll
    for (int i = 0; i < PER_THREAD; ++i) {
      const int id = tid + i * NT;
      const int row = row0 + id / CH;
      const int c = id % CH;
      if (row < N) {
        r[i] = *reinterpret_cast<const uint4*>(base + (size_t)row * D + c * 8);
      } else {
        r[i] = make_uint4(0, 0, 0, 0);
      }
    }
  }
  __device__ __forceinline__ void store(char* lds, int tid) const {
#pragma unroll
    for (int i = 0; i < PER_THREAD; ++i) {
      const int id = tid + i * NT;
      *reinterpret_cast<uint4*>(lds + tile_off<D>(id / CH, id % CH)) = r[i];
    }
  }
};

// Row fragment: lane l gets T[r0 + l%32][16*kk + 8*(l/32) .. +7] (an A or B
// operand whose contraction runs along d). `roff` is the lane's precomputed
// tile_off for chunk 2*kk + l/32 of its row, see RowFrag.
__device__ __forceinline__ bf16x8 lds_frag_row(const char* lds, int off) {
  return as_bf16x8(*reinterpret_cast<const uint4*>(lds + off));
}

// Per-lane offsets of the row fragments of rows r0 + l%32 (r0 a multiple of
// 32, added by the caller as r0 * 2D), for every kk = 0 .. D/16 - 1.
template <int D>
struct RowFrag {
  int off[D / 16];
  __device__ __forceinline__ void init(int lane) {
    const int row = lane & 31, h = lane >> 5;
#pragma unroll
    for (int kk = 0; kk < D / 16; ++kk) off[kk] = tile_off<D>(row, 2 * kk + h);
  }
};

// Same offsets from one register: chunk 2*kk + h of a row swizzled by s is
// 2*kk ^ (h ^ s) (2*kk is even and h < 2), and the row term only has bits
// above the chunk bits, so the offset of step kk is base ^ (32 * kk).
template <int D>
struct RowFragX {
  int base;
  __device__ __forceinline__ void init(int lane) { base = tile_off<D>(lane & 31, lane >> 5); }
  __device__ __forceinline__ int off(int kk) const { return base ^ (32 * kk); }
};

// Transposed fragment: operand whose contraction runs along rows. For
// contraction step base row k0 (a multiple of 16) and column block c0 (a
// multiple of 32), lane l gets T[k0 + 8*(t/4) + 4*(l/32) + t%4][c0 + l%32]
// in slot t = 0..7 — the row order of an accumulator reused as an operand.
// Built from two ds_read_b64_tr_b16: within each 16-lane group, lane i of the
// result takes element i%4 of the 8 bytes addressed by lane 4e + i/4 of the
// group, for e = 0..3.
template <int D>
struct TrFrag {
  int off[2][D / 32];  // [read][column block]
  __device__ __forceinline__ void init(int lane) {
    const int g = lane >> 4, j = lane & 15;
#pragma unroll
    for (int rd = 0; rd < 2; ++rd) {
      const int row = 8 * rd + 4 * (g >> 1) + (j >> 2);
#pragma unroll
      for (int cb = 0; cb < D / 32; ++cb) {
        const int col = 32 * cb + 16 * (g & 1) + 4 * (j & 3);
        off[rd][cb] = row * (2 * D) + 16 * ((col >> 3) ^ swz<D>(row)) + 2 * (col & 7);
      }
    }
  }
  // k0: contraction base row (multiple of 16); the row part of the swizzle
  // depends only on the low 4 row bits, so k0 enters as a plain offset.
  __device__ __forceinline__ bf16x8 load(const char* lds, int k0, int cb) const {
    const char* p0 = lds + k0 * (2 * D) + off[0][cb];
    const char* p1 = lds + k0 * (2 * D) + off[1][cb];
    bf16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(p0));
    bf16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(p1));
    bf16x8 r;
    r[0] = lo[0]; r[1] = lo[1]; r[2] = lo[2]; r[3] = lo[3];
    r[4] = hi[0]; r[5] = hi[1]; r[6] = hi[2]; r[7] = hi[3];
    return r;
  }
};

// TrFrag with two offset registers: column block cb moves the chunk index
// by 4*cb, which lies in chunk bits the row swizzle XORs but no other term
// of the offset touches, so the offset for cb is off[read] ^ (64 * cb).
template <int D>
struct TrFragX {
  int off[2];
  __device__ __forceinline__ void init(int lane) {
    TrFrag<D> t;
    t.init(lane);
    off[0] = t.off[0][0];
    off[1] = t.off[1][0];
  }
  __device__ __forceinline__ bf16x8 load(const char* lds, int k0, int cb) const {
    const char* p0 = lds + k0 * (2 * D) + (off[0] ^ (64 * cb));
    const char* p1 = lds + k0 * (2 * D) + (off[1] ^ (64 * cb));
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

// Direct global -> LDS copy of an R x D bf16 tile (rows row0 .. row0+R-1 of
// a [N][D] matrix behind `r`) into the swizzled layout of tile_off. One
// wave instruction fills 1 KB of consecutive LDS (16 bytes per lane), so
// each lane fetches the chunk whose swizzled home is its LDS slot. Rows past
// the end read as zeros. The NW waves of the group split the instructions.
template <int D, int R, int NW>
struct TileDma {
  static constexpr int CH = D / 8;
  static constexpr int INSTR = R * CH / 64;  // wave instructions per tile
  static constexpr int PER_WAVE = INSTR >= NW ? INSTR / NW : 1;
  static_assert(INSTR % NW == 0 || NW % INSTR == 0, "tile must divide evenly among waves");
  static constexpr bool ALL_ACTIVE = INSTR >= NW;  // every wave has a share
  int voff[PER_WAVE];  // byte offset of this lane's chunk relative to row0
  int lds_off;         // LDS byte offset of this wave's first instruction
  bool active;         // false for waves left without work on small tiles

  __device__ __forceinline__ void init(int wave, int lane) {
#pragma unroll
    for (int i = 0; i < PER_WAVE; ++i) {
      const int gi = (wave * PER_WAVE + i) % INSTR;
      const int pos = gi * 64 + lane;  // 16-byte slot in the tile
      const int row = pos / CH, pc = pos % CH;
      voff[i] = row * (2 * D) + 16 * (pc ^ swz<D>(row));
    }
    lds_off = (wave * PER_WAVE) % INSTR * 1024;
    active = wave * PER_WAVE < INSTR;
  }
  // Instruction i (< PER_WAVE) of this wave's share of the tile.
  __device__ __forceinline__ void issue_one(rsrc_t r, int row0, char* lds_tile, int i) const {
    if (!ALL_ACTIVE && !active) return;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void_t*)(lds_tile + lds_off + i * 1024), 16,
                                             row0 * (2 * D) + voff[i], 0, 0, 0);
  }
  __device__ __forceinline__ void issue(rsrc_t r, int row0, char* lds_tile) const {
    if (!ALL_ACTIVE && !active) return;
    const int base = row0 * (2 * D);
#pragma unroll
    for (int i = 0; i < PER_WAVE; ++i)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void_t*)(lds_tile + lds_off + i * 1024), 16, base + voff[i], 0,
                                               0, 0);
  }
};

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
