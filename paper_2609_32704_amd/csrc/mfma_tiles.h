// Shared building blocks of the matrix-core kernels (gfx950).
//
// * bf16 row-major tiles in LDS with 16-byte chunks XOR-swizzled by row, so
//   that 16 lanes reading the same chunk of 16 consecutive rows, or the
//   transposing reads below, touch distinct banks;
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

// A swizzled tile of ROWS rows x D bf16 columns (row pitch 2 D bytes).
template <int D, int ROWS>
struct SwzTile {
  static constexpr int CH = D / 8;             // 16-byte chunks per row
  static constexpr int BYTES = ROWS * D * 2;
  static constexpr int LOADS = BYTES / 1024;   // 1 KB direct loads per tile
  __device__ static inline int off(int row, int chunk) { return row * (D * 2) + ((chunk ^ (row % CH)) << 4); }
  // byte address of the 8-byte group holding column col (a multiple of 4)
  __device__ static inline int off_col(int row, int col) { return off(row, col >> 3) + ((col & 7) << 1); }
};

// Copy rows [first, first + ROWS) of a row-major [n_rows][D] bf16 matrix into
// a swizzled LDS tile; rows past n_rows repeat row n_rows - 1 (callers mask
// them).  Every wave of the workgroup takes every nw-th 1 KB piece.
template <int D, int ROWS>
__device__ inline void load_tile(const __bf16* base, int64_t first, int64_t n_rows, unsigned char* lds, int wave,
                                 int nw, int lane) {
  using T = SwzTile<D, ROWS>;
  for (int n = wave; n < T::LOADS; n += nw) {
    const int flat = n * 64 + lane;  // 16-byte unit index == LDS position
    const int row = flat / T::CH, slot = flat % T::CH;
    const int chunk = slot ^ (row % T::CH);
    int64_t r = first + row;
    if (r >= n_rows) r = n_rows - 1;
    __builtin_amdgcn_global_load_lds(reinterpret_cast<const void*>(base + r * D + chunk * 8),
                                     (lds_void*)(lds + n * 1024), 16, 0, 0);
  }
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

// s_waitcnt immediate that waits until at most n (< 64) vector-memory
// operations are outstanding and leaves the other counters alone (gfx9 layout:
// vmcnt bits 3:0 and 15:14, expcnt 6:4, lgkmcnt 11:8).
constexpr int vmcnt_only(int n) { return (n & 15) | ((n >> 4) << 14) | (7 << 4) | (15 << 8); }

__device__ inline f32x4 mfma16(const bf16x8& a, const bf16x8& b, const f32x4& c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

}  // namespace cowa
