// Device helpers shared by the fused forward kernel and the layer-by-layer operators (gfx950):
// vector types, bf16 packing, vmcnt waits, buffer loads that write LDS directly, the LDS swizzles of
// K and V tiles and the loader that moves such tiles. Internal; included by the kernel sources only.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace fa {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;

constexpr int kNumXcd = 8;

// Row order of a 32-key block in the score product's A operand: A-row i holds key perm32(i).
// With the 32x32 accumulator layout (register r of a lane in half h holds A-row
// 8*(r/4) + 4*h + r%4), register r then holds key 16*(r/8) + 8*h + r%8.
__device__ __forceinline__ int perm32(int i) { return (i & ~12) | ((i & 4) << 1) | ((i & 8) >> 1); }

// LDS on gfx950 has 64 four-byte banks (256 bytes per cycle). A ds_read_b128 is served 16 lanes per
// cycle and a ds_read_b64_tr_b16 32 lanes per cycle; the lanes served together must touch 16
// different 16-byte bank slots to avoid conflicts.
//
// XOR swizzle of the 16-byte chunks of K-tile row `row`, as a function of the reading lane
// i = perm32(row % 32) (lanes 16m..16m+15 of a K fragment read rows perm32(i) of one chunk column).
// DQK = 128 (16 chunks per row, every row starts at bank 0): a 4-bit XOR by i. DQK = 64 or 192 (rows
// start alternately at bank 0 and 32, i.e. row parity = i parity selects the half): a 3-bit XOR by
// i / 2, which stays inside each aligned group of 8 chunks.
template <int DQK>
__device__ __forceinline__ int k_lane_swizzle(int i) { return (DQK / 8) % 16 == 0 ? (i & 15) : ((i >> 1) & 7); }
template <int DQK>
__device__ __forceinline__ int k_swizzle(int row) { return k_lane_swizzle<DQK>(perm32(row & 31)); }

// XOR swizzle of the 16-byte chunks of V-tile row `key`. Lanes 0..31 of the transpose read touch
// keys k..k+3 (k a multiple of 4), 64 bytes each, at the same chunk columns: DV = 128 spreads the
// four rows over chunk bits 2..3 (every row starts at bank 0); DV = 64 over bits 1..2 (there row
// parity already separates bank halves).
template <int DV>
__device__ __forceinline__ int v_swizzle(int key) { return DV >= 128 ? 4 * (key & 3) : 2 * (key & 3); }

template <class T, class U>
__device__ __forceinline__ T bit_cast(const U& u) {
  static_assert(sizeof(T) == sizeof(U), "size mismatch");
  return __builtin_bit_cast(T, u);
}

// max / sum of a per-lane value with the value of the lane 32 positions away. After
// permlane32_swap(x, x) the two results hold {own, partner} in some order on every lane, and both
// reductions are symmetric.
__device__ __forceinline__ float half_swap_max(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float half_swap_sum(float x) {
  auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  f32x2 f = {lo, hi};
  return bit_cast<uint32_t>(__builtin_convertvector(f, bf16x2));  // v_cvt_pk_bf16_f32, RNE
}

// Wait until at most N vector-memory instructions of this wave are outstanding (vmcnt only).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

// One 64-lane buffer load of 16 bytes per lane that writes LDS directly: LDS bytes
// [lds, lds + 1024) receive the lanes' 16 bytes in lane order; lane bytes [voff, voff + 16) of the
// buffer described by `rsrc` (raw: base, num_records in bytes). Lanes whose range lies past
// num_records receive zeros. Issued as inline asm so that the compiler does not track it: it would
// otherwise assume that any later LDS read may alias the in-flight load and wait for every
// outstanding load first. Completion is ordered explicitly instead (vmcnt wait on the issuing wave,
// then a workgroup barrier) before any wave reads the destination. The SALU write of M0 needs one
// wait state before the load.
__device__ __forceinline__ void dma16_buffer(u32x4 rsrc, uint32_t voff, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tbuffer_load_dwordx4 %0, %1, 0 offen lds"
               :
               : "v"(voff), "s"(rsrc), "s"(lds)
               : "memory", "m0");
}
__device__ __forceinline__ uint32_t lds_offset(const void* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
}
// Compiler-level memory fence (no instruction): keeps LDS reads on their side of a barrier.
__device__ __forceinline__ void compiler_fence() { asm volatile("" : : : "memory"); }

// This wave's share of the direct-to-LDS loads of one K or V tile (BN rows of CH 16-byte chunks).
// Physical chunk p of a slot holds logical chunk (p % CH) ^ swz(row) of row p / CH, so the lanes'
// source offsets carry the swizzle; they are computed once. Each tile is described by a buffer
// whose base is the tile's first row and whose size ends at the workgroup's last visible key
// (Sk, or the causal limit of its last query row): rows past it load as zeros without a memory
// access (their scores are masked and their V rows meet P = 0), which also makes the loads of tiles
// past the last one cheap. One head's K or V spans less than 4 GiB (the API bounds Sk * d), so
// 32-bit record counts suffice.
template <int NWAVES, int BN, int CH>
struct TileLoader {
  static constexpr int NI = BN * CH / 64 / NWAVES;  // loads per wave per tile
  static constexpr uint32_t kRowBytes = CH * 16;
  uint64_t head;      // first row of this head (wave-uniform)
  uint32_t rows;      // keys visible to the workgroup
  uint32_t voff[NI];  // bytes from the tile's first row
  template <class Swz>
  __device__ __forceinline__ void init(const uint16_t* head_, int nrows, int wave, int lane, Swz swz) {
    head = reinterpret_cast<uint64_t>(head_);
    rows = (uint32_t)nrows;
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int pch = (wave * NI + i) * 64 + lane;
      const int row = pch / CH;
      voff[i] = (uint32_t)(row * CH + ((pch % CH) ^ swz(row))) * 16u;
    }
  }
  // Buffer of the tile whose first row is key n0 (n0 >= 0; a tile at or past Sk gets an empty
  // buffer and loads zeros), and this wave's LDS base in `slot`.
  __device__ __forceinline__ u32x4 rsrc(int n0) const {
    const uint64_t base = head + (uint64_t)n0 * kRowBytes;
    const uint32_t left = (int)rows > n0 ? (rows - (uint32_t)n0) * kRowBytes : 0u;
    return u32x4{(uint32_t)base, (uint32_t)(base >> 32) & 0xffffu, left, 0x00020000u};
  }
  // Walking the tiles in order: rsrc_walk(n0, rem) is rsrc(n0) with rem = rows - n0 (signed, may be
  // negative), and advance() moves both on by BN rows. The base's high word gains only the carry (a
  // device address stays below 2^48, so the stride field above bit 16 stays 0), and the bytes left
  // are max(rem, 0) rows: scalar add, add-with-carry, max and shift, where rsrc() multiplies and
  // compares. A saturating unsigned subtract instead would be selected as a vector instruction, and
  // the descriptor must stay in scalar registers.
  __device__ __forceinline__ u32x4 rsrc_walk(int n0, int& rem) const {
    rem = (int)rows - n0;
    return rsrc(n0);
  }
  __device__ __forceinline__ void advance(u32x4& r, int& rem) const {
    constexpr uint32_t kStep = BN * kRowBytes;
    const uint64_t base = (((uint64_t)r.y << 32) | r.x) + kStep;
    r.x = (uint32_t)base;
    r.y = (uint32_t)(base >> 32);
    rem -= BN;
    r.z = (uint32_t)max(rem, 0) * kRowBytes;
  }
  __device__ __forceinline__ uint32_t lds(unsigned char* slot, int wave) const {
    return lds_offset(slot + wave * NI * 1024);
  }
  __device__ __forceinline__ void issue_one(const u32x4& r, uint32_t l, int i) const {
    dma16_buffer(r, voff[i], l + i * 1024);
  }
  // Issue all loads of the tile at key n0 into `slot` at once.
  __device__ __forceinline__ void issue(int n0, unsigned char* slot, int wave) const {
    const u32x4 r = rsrc(n0);
    const uint32_t l = lds(slot, wave);
#pragma unroll
    for (int i = 0; i < NI; ++i) issue_one(r, l, i);
  }
};

}  // namespace
}  // namespace fa
