// Shared building blocks of the matrix-core kernels (gfx950).
//
// * bf16 row-major tiles in LDS with 16-byte chunks XOR-swizzled by row (see
//   swz below), so that every read pattern of the kernels (row fragments by
//   ds_read_b128, the transposing reads below) is free of bank conflicts;
// * direct global -> LDS copies of such tiles (global_load_lds, 16 bytes per
//   lane: lane l of one instruction lands at LDS base + 16 l);
// * transposing LDS reads (ds_read_b64_tr_b16).  Within each group of 16
//   lanes, lane s supplies the address of 4 consecutive bf16 values and output
//   lane j receives value j % 4 of the lanes j / 4, 4 + j / 4, 8 + j / 4 and
//   12 + j / 4.  With lane s pointing at row r0 + s / 4, column c0 + 4 (s % 4)
//   of a row-major tile, output lane j holds column c0 + j of rows r0 .. r0+3:
//   the k-major MFMA operand of a transposed tile.
// * the XCD-aware workgroup order.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>
#include <utility>

namespace cowa {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

// Workgroups id, id + 8, id + 16, ... land on the same XCD (round-robin
// dispatch over the 8 XCDs).  Hand each XCD whole chunks of 8 consecutive work
// items so that items sharing K/V or Q/dO blocks share that XCD's L2.
__device__ inline int xcd_remap(int id, int total) {
  const int full = (total / 64) * 64;
  if (id >= full) return id;
  const int xcd = id & 7, slot = id >> 3;
  const int chunk = (slot >> 3) * 8 + xcd;
  return chunk * 8 + (slot & 7);
}

// Workgroup id -> (row, group, unit) for a grid of n_rows x units x groups
// workgroups, where the groups of one unit (one sequence and KV head) and
// neighbouring rows read nearly the same K/V (or Q/dO) blocks.  Work is cut into
// clusters of cq consecutive rows x the groups of one unit; cluster c runs on
// XCD c % 8, so the workgroups an XCD runs together (one cluster) share its L2.
// Rows go out first to last, or last to first (descending), whole cluster rows
// at a time; the unit of an XCD's cluster rotates from one row range to the
// next, so every XCD gets the same mix of units.  Shapes that do not tile this
// way use the row order with chunks of 8 consecutive items per XCD.
struct WorkItem {
  int row, group, unit;
};
__device__ inline WorkItem cluster_item(int id, int n_rows, int groups, int units, int cq, bool descending) {
  WorkItem w;
  const int n_clusters = units * (n_rows / cq);
  if (n_rows % cq == 0 && n_clusters % 8 == 0) {
    const int cs = cq * groups;  // workgroups per cluster
    const int xcd = id & 7, n = id >> 3;
    const int c = (n / cs) * 8 + xcd, item = n % cs;
    const int r = c / units;
    w.unit = (c % units + r) % units;
    w.group = item % groups;
    w.row = r * cq + item / groups;
  } else {
    const int per_row = groups * units;
    const int work = xcd_remap(id, n_rows * per_row);
    w.row = work / per_row;
    w.unit = (work % per_row) / groups;
    w.group = work % groups;
  }
  if (descending) w.row = n_rows - 1 - w.row;
  return w;
}

// Rows per cluster for cluster_item: at most cq_max, halved (down to 4) until
// there are at least 16 clusters per XCD.  The dispatcher hands workgroup ids to
// the XCDs round-robin, so each XCD takes a fixed share of the clusters; rows of
// unequal length (at one end of a sequence only some rows reach a long-range
// window or the sink) must spread over many clusters to load every XCD alike
// when there are few units (one KV head on a device, one short sequence).
__device__ inline int cluster_rows(int n_rows, int units, int cq_max) {
  int cq = cq_max;
  while (cq > 4 && (int64_t)units * (n_rows / cq) < 8 * 16) cq >>= 1;
  return cq;
}

// XOR applied to the 16-byte chunk index of a row; depends on row % 16 only.
// The gfx950 LDS has 64 four-byte banks (256 bytes per clock).  Measured with
// bank-conflict counters: ds_read_b128 serves 16 lanes per clock, in the
// groups {0-3, 12-15, 20-23, 24-27} and {4-11, 16-19, 28-31} (and the same
// +32), i.e. lanes with equal lane / 32 and equal parity of bits 2..4 of the
// lane; ds_read_b64 and ds_read_b64_tr_b16 serve lanes 0-31, then 32-63.  A
// read is conflict-free iff the lanes served together touch distinct banks.
// The masks below were found by exhaustive search over that model so that
// every read pattern of the kernels is conflict-free (D = 128 and D = 64):
//  * row fragments: rows r .. r+15 (r a multiple of 16), lane l reading row
//    r + l % 16 and chunk 4 ks + l / 16 (backward and dQ pass), or rows
//    r .. r+31, lane l reading row r + l % 32 and chunk 2 ks + l / 32 (forward);
//  * transposing reads of 4 rows x 2 chunks per 16 lanes (tr8_off below) and
//    the forward's V^T reads (rows 4 (l / 32) + (l % 16) / 4 (+ 8), columns
//    32 md + 16 ((l / 16) % 2) + 4 (l % 4)).
// Bits 1..0 of both masks are the same function of row / 4: 0, 2, 3, 1.
template <int CH>
__host__ __device__ inline int swz(int row) {
  static_assert(CH == 8 || CH == 16, "head_dim 64 or 128");
  const int hi = ((((row >> 2) ^ (row >> 3)) & 1) << 1) | ((row >> 3) & 1);
  if constexpr (CH == 16) return ((row & 3) << 2) | hi;
  return (((row >> 1) & 1) << 2) | hi;
}

// A swizzled tile of ROWS rows x D bf16 columns (row pitch 2 D bytes).
template <int D, int ROWS>
struct SwzTile {
  static constexpr int CH = D / 8;             // 16-byte chunks per row
  static constexpr int BYTES = ROWS * D * 2;
  static constexpr int LOADS = BYTES / 1024;   // 1 KB direct loads per tile
  __device__ static inline int off(int row, int chunk) { return row * (D * 2) + ((chunk ^ swz<CH>(row)) << 4); }
  // byte address of the 8-byte group holding column col (a multiple of 4)
  __device__ static inline int off_col(int row, int col) { return off(row, col >> 3) + ((col & 7) << 1); }
};

// Copy rows [first, first + ROWS) of a row-major [n_rows][D] bf16 matrix into
// a swizzled LDS tile; rows past n_rows repeat row n_rows - 1 (callers mask
// them).  The NW waves of the workgroup take the 1 KB pieces in turn; wave must
// be wave-uniform.  Since NW pieces span a multiple of 16 rows, a lane's row
// modulo 16, and so its swizzled chunk, is the same in every piece it copies.
template <int D, int ROWS, int NW>
__device__ inline void load_tile(const __bf16* base, int first, int n_rows, unsigned char* lds, int wave, int lane) {
  using T = SwzTile<D, ROWS>;
  constexpr int RPL = 1024 / (D * 2);  // rows per piece
  static_assert(T::LOADS % NW == 0 && (NW * RPL) % 16 == 0, "piece layout");
  const int row0 = wave * RPL + lane / T::CH;
  const int col = (((lane % T::CH) ^ swz<T::CH>(row0)) << 3);
#pragma unroll
  for (int n = 0; n < T::LOADS / NW; ++n) {
    int r = first + n * NW * RPL + row0;
    r = r < n_rows ? r : n_rows - 1;
    __builtin_amdgcn_global_load_lds(reinterpret_cast<const void*>(base + (int64_t)r * D + col),
                                     (lds_void*)(lds + (n * NW + wave) * 1024), 16, 0, 0);
  }
}

// Global -> LDS copies issued as inline assembly: 16 (dma16) or 4 (dma4) bytes
// per lane, lane l landing at LDS byte address lds_base + 16 l (or 4 l).  The
// compiler does not see these as memory operations, so it neither counts them
// in its own s_waitcnt arithmetic nor makes unrelated LDS reads wait for them;
// the caller waits for them explicitly (s_waitcnt vmcnt) before their data is
// read and before the LDS they target is reused.  lds_base must be uniform.
// Each copy sets M0 (the LDS destination) itself.  The compiler warns that it
// may not preserve a reserved register named as clobbered; for gfx950 it keeps
// no value of its own in M0 in these kernels (every M0 write in their device
// assembly comes from these statements), so nothing live is overwritten.
__device__ inline uint32_t lds_addr(const unsigned char* p) {
  return (uint32_t)(uintptr_t)(lds_void*)p;
}
__device__ inline void dma16(const void* gptr, uint32_t lds_base) {
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off"
               :
               : "v"(gptr), "s"(lds_base)
               : "memory", "m0");
}
__device__ inline void dma4(const void* gptr, uint32_t lds_base) {
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dword %0, off"
               :
               : "v"(gptr), "s"(lds_base)
               : "memory", "m0");
}

typedef int i32x4 __attribute__((ext_vector_type(4)));

// Raw buffer resource over [base, base + bytes) (GFX9 layout, stride 0): loads
// at offsets past `bytes` return zero instead of touching memory.
__device__ inline i32x4 buffer_rsrc(const void* base, uint32_t bytes) {
  const uint64_t a = (uint64_t)base;
  return i32x4{(int)(uint32_t)a, (int)((a >> 32) & 0xffffu), (int)bytes, 0x00020000};
}
// 16 bytes per lane from a buffer straight into LDS: lane l lands at
// lds_base + 16 l.  Issued as assembly and waited for explicitly, like dma16.
__device__ inline void dma16_buf(uint32_t voff, i32x4 rsrc, uint32_t lds_base) {
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tbuffer_load_dwordx4 %0, %1, 0 offen lds"
               :
               : "v"(voff), "s"(rsrc), "s"(lds_base)
               : "memory", "m0");
}

// load_tile through dma16 (same layout and piece order).
template <int D, int ROWS, int NW>
__device__ inline void load_tile_asm(const __bf16* base, int first, int n_rows, uint32_t lds, int wave, int lane) {
  using T = SwzTile<D, ROWS>;
  constexpr int RPL = 1024 / (D * 2);
  static_assert(T::LOADS % NW == 0 && (NW * RPL) % 16 == 0, "piece layout");
  const int row0 = wave * RPL + lane / T::CH;
  const int col = (((lane % T::CH) ^ swz<T::CH>(row0)) << 3);
#pragma unroll
  for (int n = 0; n < T::LOADS / NW; ++n) {
    int r = first + n * NW * RPL + row0;
    r = r < n_rows ? r : n_rows - 1;
    dma16(base + (int64_t)r * D + col, __builtin_amdgcn_readfirstlane(lds + (n * NW + wave) * 1024));
  }
}

// load_tile_asm for a wave-uniform wave count known at run time.
template <int D, int ROWS>
__device__ inline void load_tile_asm_nw(const __bf16* base, int first, int n_rows, uint32_t lds, int wave, int nw,
                                        int lane) {
  using T = SwzTile<D, ROWS>;
  constexpr int RPL = 1024 / (D * 2);
  if constexpr (T::LOADS % 8 == 0 && (8 * RPL) % 16 == 0) {
    if (nw == 8) return load_tile_asm<D, ROWS, 8>(base, first, n_rows, lds, wave, lane);
  }
  if constexpr (T::LOADS % 4 == 0 && (4 * RPL) % 16 == 0) {
    if (nw == 4) return load_tile_asm<D, ROWS, 4>(base, first, n_rows, lds, wave, lane);
  }
  for (int n = wave; n < T::LOADS; n += nw) {
    const int flat = n * 64 + lane;
    const int row = flat / T::CH, slot = flat % T::CH;
    const int chunk = slot ^ swz<T::CH>(row);
    int r = first + row;
    r = r < n_rows ? r : n_rows - 1;
    dma16(base + (int64_t)r * D + chunk * 8, __builtin_amdgcn_readfirstlane(lds + n * 1024));
  }
}

// The same for any wave count (a lane's chunk recomputed per piece).
template <int D, int ROWS>
__device__ inline void load_tile_any(const __bf16* base, int first, int n_rows, unsigned char* lds, int wave, int nw,
                                     int lane) {
  using T = SwzTile<D, ROWS>;
  for (int n = wave; n < T::LOADS; n += nw) {
    const int flat = n * 64 + lane;  // 16-byte unit index == LDS position
    const int row = flat / T::CH, slot = flat % T::CH;
    const int chunk = slot ^ swz<T::CH>(row);
    int r = first + row;
    r = r < n_rows ? r : n_rows - 1;
    __builtin_amdgcn_global_load_lds(reinterpret_cast<const void*>(base + (int64_t)r * D + chunk * 8),
                                     (lds_void*)(lds + n * 1024), 16, 0, 0);
  }
}

// Dispatch on a wave-uniform wave count.
template <int D, int ROWS>
__device__ inline void load_tile_nw(const __bf16* base, int first, int n_rows, unsigned char* lds, int wave, int nw,
                                    int lane) {
  using T = SwzTile<D, ROWS>;
  constexpr int RPL = 1024 / (D * 2);
  if constexpr (T::LOADS % 8 == 0 && (8 * RPL) % 16 == 0) {
    if (nw == 8) return load_tile<D, ROWS, 8>(base, first, n_rows, lds, wave, lane);
  }
  if constexpr (T::LOADS % 4 == 0 && (4 * RPL) % 16 == 0) {
    if (nw == 4) return load_tile<D, ROWS, 4>(base, first, n_rows, lds, wave, lane);
  }
  load_tile_any<D, ROWS>(base, first, n_rows, lds, wave, nw, lane);
}

// 16-byte row fragment: row `row`, columns 8 chunk .. 8 chunk + 7.
template <int D, int ROWS>
__device__ inline bf16x8 read_row8(const unsigned char* tile, int row, int chunk) {
  return *reinterpret_cast<const bf16x8*>(tile + SwzTile<D, ROWS>::off(row, chunk));
}

// Transposed MFMA operand from a row-major swizzled tile: output lane j of each
// 16-lane group gets column c0 + j of rows r0 + 4 g + t (t = 0..3) in its
// first four slots and of rows r0 + 16 + 4 g + t in the last four, g = lane / 16.
template <int D, int ROWS>
__device__ inline bf16x8 read_tr8(const unsigned char* tile, int r0, int c0, int lr, int lg) {
  using T = SwzTile<D, ROWS>;
  const int row = r0 + 4 * lg + (lr >> 2);
  const int col = c0 + 4 * (lr & 3);
  const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(tile + T::off_col(row, col)));
  const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(tile + T::off_col(row + 16, col)));
  const bf16x4 a = __builtin_bit_cast(bf16x4, lo), b = __builtin_bit_cast(bf16x4, hi);
  return bf16x8{a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
}

// Same from a plain (unswizzled) row-major tile with a row pitch in bytes.
__device__ inline bf16x8 read_tr8_plain(const unsigned char* tile, int pitch, int r0, int c0, int lr, int lg) {
  const int row = r0 + 4 * lg + (lr >> 2);
  const int col = c0 + 4 * (lr & 3);
  const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(tile + row * pitch + col * 2));
  const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(tile + (row + 16) * pitch + col * 2));
  const bf16x4 a = __builtin_bit_cast(bf16x4, lo), b = __builtin_bit_cast(bf16x4, hi);
  return bf16x8{a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
}

// Per-lane byte offsets of the two read patterns, for rows 0..15 of a tile;
// since the swizzle depends on row % 16, rows 16 m + ... add 16 m D 2 bytes
// (a constant the compiler folds into the instruction's offset field).
//  row fragment: lane (lr, lg) reads row lr, chunk 4 ks + lg;
template <int D>
__device__ inline int row8_off(int lr, int lg, int ks) {
  return lr * (D * 2) + (((4 * ks + lg) ^ swz<D / 8>(lr)) << 4);
}
//  transposing read: lane (lr, lg) points at row 4 lg + lr / 4, column 16 md + 4 (lr % 4).
template <int D>
__device__ inline int tr8_off(int lr, int lg, int md) {
  const int row = 4 * lg + (lr >> 2), col = 16 * md + 4 * (lr & 3);
  return row * (D * 2) + (((col >> 3) ^ swz<D / 8>(row)) << 4) + ((col & 7) << 1);
}
__device__ inline bf16x8 ld_row8(const unsigned char* p) { return *reinterpret_cast<const bf16x8*>(p); }
// the transposed operand of rows r0 .. r0+31 (p at row r0 of the pattern above;
// row_bytes = 2 D): rows r0 + 4 g + t in slots 0..3, rows r0 + 16 + 4 g + t in 4..7
__device__ inline bf16x8 ld_tr8(const unsigned char* p, int row_bytes) {
  const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)p);
  const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(p + 16 * row_bytes));
  const bf16x4 a = __builtin_bit_cast(bf16x4, lo), b = __builtin_bit_cast(bf16x4, hi);
  return bf16x8{a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
}

// s_waitcnt immediate that waits until at most n (< 64) vector-memory
// operations are outstanding and leaves the other counters alone (gfx9 layout:
// vmcnt bits 3:0 and 15:14, expcnt 6:4, lgkmcnt 11:8).
constexpr int vmcnt_only(int n) { return (n & 15) | ((n >> 4) << 14) | (7 << 4) | (15 << 8); }

// f(std::integral_constant<int, I>) for I = 0 .. N-1, expanded at compile time
// (a fixed instruction schedule whose steps differ by their index).
template <class F, int... I>
__device__ inline void static_for_impl(F&& f, std::integer_sequence<int, I...>) {
  (f(std::integral_constant<int, I>{}), ...);
}
template <int N, class F>
__device__ inline void static_for(F&& f) {
  static_for_impl(f, std::make_integer_sequence<int, N>{});
}

__device__ inline f32x4 mfma16(const bf16x8& a, const bf16x8& b, const f32x4& c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

}  // namespace cowa
