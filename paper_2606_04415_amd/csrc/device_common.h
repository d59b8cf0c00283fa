// Device helpers shared by the attention kernels (gfx950, wave64).
//
// Matrix-core convention used throughout (v_mfma_f32_16x16x32_bf16): a wave
// computes D[16][16] += A[16][32] * B[32][16]. Lane l = 16*g + n supplies row
// n of A and column n of B, each as 8 bf16 covering the 8 contraction slots
// of lane group g; it receives D[4*g + r][n] for r = 0..3. Which contraction
// index sits in which slot does not matter as long as A and B use the same
// slots, which lets the kernels permute the contraction (head dims for QK^T,
// keys for PV) freely.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace flexattn {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

__device__ __forceinline__ f32x4 mfma_16x16x32(const u32x4& a, const u32x4& b, const f32x4& c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, a),
                                                 __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

__device__ __forceinline__ u32x4 zero4() { return u32x4{0u, 0u, 0u, 0u}; }

// s_waitcnt with only the vector-memory counter constrained (gfx9 encoding:
// vmcnt bits [3:0] and [15:14], expcnt [6:4] = 7, lgkmcnt [11:8] = 15).
template <int N>
__device__ __forceinline__ void wait_vmem() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | 0x0F70);
}
// Work-group barrier for LDS hand-offs that leaves vector-memory loads in
// flight: this wave's LDS writes complete (lgkmcnt 0), then s_barrier. (The
// fence inside __syncthreads also waits for every outstanding global load,
// which would drain a prefetch pipeline at each tile.) The signal fences keep
// the compiler from moving LDS accesses across it.
__device__ __forceinline__ void lds_barrier() {
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
  __builtin_amdgcn_s_waitcnt(0xC07F);   // vmcnt 63, expcnt 7, lgkmcnt 0
  __builtin_amdgcn_s_barrier();
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

// Order one wave's LDS accesses around an exchange between its own lanes: a
// wave's LDS instructions execute in issue order, so the barrier only has to
// stop the compiler from moving accesses across it.
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// Word idx of an array the kernel only reads, through a scalar load (the
// index is made wave-uniform): scalar loads are counted apart from vector
// memory, so reading plan metadata does not wait for the K/V loads in
// flight, which a vector load issued after them would (vector loads retire
// in order).
typedef const __attribute__((address_space(4))) int32_t* const_i32_ptr;
__device__ __forceinline__ int32_t scalar_word(const int32_t* base, int idx) {
  return ((const_i32_ptr)(base))[__builtin_amdgcn_readfirstlane(idx)];
}

// Let every outstanding vector-memory access land (placed after loads issued
// before a pipelined loop, so loop-carried wait tracking starts clean).
__device__ __forceinline__ void wait_vmem_all() { wait_vmem<0>(); }

// Pack two floats into two bf16 (round to nearest even) in one dword, lo first.
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{lo, hi}, bf16x2));
}

// Word 3 of a raw (unswizzled, stride 0) buffer resource on gfx9: 32-bit
// data format, so out-of-range dword loads return zero.
constexpr int kBufferFlags = 0x00020000;

// Element offset of (page, slot, head) in a paged cache with element strides.
struct PagedCache {
  const uint16_t* base;
  int64_t sp, ss, sh;
  __device__ __forceinline__ const uint16_t* row(int32_t page, int32_t slot, int32_t head) const {
    return base + int64_t(page) * sp + int64_t(slot) * ss + int64_t(head) * sh;
  }
};

// Physical page of key t of a sequence whose block-table row is bt_row.
__device__ __forceinline__ int32_t page_of(const int32_t* __restrict__ bt_row, int32_t t, int32_t P) {
  return bt_row[t / P];
}

__device__ __forceinline__ u32x4 load16(const uint16_t* p) {
  return *reinterpret_cast<const u32x4*>(p);
}
__device__ __forceinline__ u32x2 load8(const uint16_t* p) {
  return *reinterpret_cast<const u32x2*>(p);
}

// ds_read_b64_tr_b16: within each group of 16 lanes, lane j supplies the LDS
// address of 4 consecutive bf16; lane i receives element i%4 of the rows that
// lanes i/4, 4 + i/4, 8 + i/4 and 12 + i/4 addressed. With lane j pointing
// at row R(j/4), column c + 4*(j%4), lane i gets column c + i of rows
// R(0..3): a B operand read straight from a row-major (key-major) tile.
typedef short v4i16 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ u32x2 lds_read_tr16(const uint16_t* lds_addr) {
  typedef __attribute__((address_space(3))) v4i16* lds_v4i16_ptr;
  const v4i16 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16_ptr)(lds_addr));
  return __builtin_bit_cast(u32x2, v);
}

// Two bf16 halves from two dwords: lo -> (x.lo, y.lo), hi -> (x.hi, y.hi)
// (one v_perm_b32 each; selector bytes 0-3 pick from x, 4-7 from y).
__device__ __forceinline__ uint32_t pair_lo(uint32_t x, uint32_t y) { return __builtin_amdgcn_perm(y, x, 0x05040100u); }
__device__ __forceinline__ uint32_t pair_hi(uint32_t x, uint32_t y) { return __builtin_amdgcn_perm(y, x, 0x07060302u); }

// 8 key rows x 8 dims (row r holds dims 0..7 of key r as 4 dwords) ->
// 8 B-operands, operand c holding dim c of keys 0..7 (dword w = keys 2w, 2w+1).
__device__ __forceinline__ void transpose8x8(const u32x4 (&rows)[8], u32x4 (&ops)[8]) {
#pragma unroll
  for (int c = 0; c < 8; ++c) {
    const int dw = c >> 1;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const uint32_t x = rows[2 * w][dw], y = rows[2 * w + 1][dw];
      ops[c][w] = (c & 1) ? pair_hi(x, y) : pair_lo(x, y);
    }
  }
}

// 8 key rows x 4 dims -> 4 B-operands (head_dim 64 layout).
__device__ __forceinline__ void transpose8x4(const u32x2 (&rows)[8], u32x4 (&ops)[4]) {
#pragma unroll
  for (int c = 0; c < 4; ++c) {
    const int dw = c >> 1;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const uint32_t x = rows[2 * w][dw], y = rows[2 * w + 1][dw];
      ops[c][w] = (c & 1) ? pair_hi(x, y) : pair_lo(x, y);
    }
  }
}

__device__ __forceinline__ float shfl_xor_f(float v, int mask) { return __shfl_xor(v, mask, 64); }
__device__ __forceinline__ float shfl_f(float v, int src) { return __shfl(v, src, 64); }

// Max / sum over the four lane groups g = 0..3 that share lane index n.
// v_permlane16_swap(x, x) returns rows (0,0,2,2) and (1,1,3,3) of x, and
// v_permlane32_swap(x, x) returns rows (0,1,0,1) and (2,3,2,3): combining
// each pair exchanges values with lane n^16, then lane n^32, on the VALU.
__device__ __forceinline__ float swap16_combine_max(float v) {
  const uint32_t u = __float_as_uint(v);
  const auto t = __builtin_amdgcn_permlane16_swap(u, u, false, false);
  return fmaxf(__uint_as_float(t[0]), __uint_as_float(t[1]));
}
__device__ __forceinline__ float swap32_combine_max(float v) {
  const uint32_t u = __float_as_uint(v);
  const auto t = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  return fmaxf(__uint_as_float(t[0]), __uint_as_float(t[1]));
}
__device__ __forceinline__ float group_max(float v) { return swap32_combine_max(swap16_combine_max(v)); }
// group_max of two values at once, in three swaps instead of four. With
// lane-group rows a = (a0..a3), b = (b0..b3): swap16(a, b) pairs a0|a1 and
// a2|a3 in rows 0 and 2 and b's in rows 1 and 3; after one max, swap32 of the
// result with itself pairs rows 0|2 and 1|3, and a last swap16 of the second
// max with itself spreads a's total to every row of one output and b's to
// every row of the other.
__device__ __forceinline__ void group_max2(float& a, float& b) {
  auto t = __builtin_amdgcn_permlane16_swap(__float_as_uint(a), __float_as_uint(b), false, false);
  const float c = fmaxf(__uint_as_float(t[0]), __uint_as_float(t[1]));
  t = __builtin_amdgcn_permlane32_swap(__float_as_uint(c), __float_as_uint(c), false, false);
  const float d = fmaxf(__uint_as_float(t[0]), __uint_as_float(t[1]));
  t = __builtin_amdgcn_permlane16_swap(__float_as_uint(d), __float_as_uint(d), false, false);
  a = __uint_as_float(t[0]);
  b = __uint_as_float(t[1]);
}
__device__ __forceinline__ float group_sum(float v) {
  uint32_t u = __float_as_uint(v);
  auto t = __builtin_amdgcn_permlane16_swap(u, u, false, false);
  v = __uint_as_float(t[0]) + __uint_as_float(t[1]);
  u = __float_as_uint(v);
  t = __builtin_amdgcn_permlane32_swap(u, u, false, false);
  return __uint_as_float(t[0]) + __uint_as_float(t[1]);
}

// Slot e (0..7) of a lane in group g within a 32-key chunk holds key
// 16*(e/4) + 4*g + (e%4): exactly the keys whose scores the lane receives from
// the two 16-key QK^T blocks, so P feeds the PV product with no data movement.
__device__ __forceinline__ int chunk_key(int e, int g) { return 16 * (e >> 2) + 4 * g + (e & 3); }

}  // namespace flexattn
