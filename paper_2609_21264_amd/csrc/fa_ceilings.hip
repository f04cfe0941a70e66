// Measured ceilings of MI355X (gfx950) for the roofline of the fused attention forward: the rate the
// matrix cores sustain on bf16 MFMAs with nothing else to do, and the clock they sustain it at; HBM
// streaming reads through VGPRs and through buffer loads that write LDS directly (the path the fused
// kernel's K/V tiles take); LDS read rates of the two read forms the fused kernel uses
// (ds_read_b128 for K fragments, ds_read_b64_tr_b16 for V fragments). These are the GPU counterparts
// of the paper's instruction-count compute ceiling and its per-level bandwidth ceilings (Sec. 5.2,
// Table 2). Built as its own library (libfa_ceilings.so); measurement only, not part of libfa.so.
//
// Every kernel records, per wave, the shader clock counter and the constant-rate real-time counter
// at its start and end (stamps[4 * wave + {0, 1, 2, 3}] = clock start, clock end, real start, real
// end), so the host can derive the sustained shader clock of the run.
//
// C ABI (all return a hipError_t value; 0 = enqueued on `stream`; hipErrorInvalidValue (1) when an
// argument is out of range, checked on the host before any launch):
//   fa_ceil_mfma(operands, out, stamps, waves_per_simd, n_wg, iters, stream)
//       n_wg workgroups of 4 * waves_per_simd waves (waves_per_simd 1 or 2), each holding 96 KiB of
//       LDS so that one workgroup occupies a CU; every wave runs iters x 16 v_mfma_f32_32x32x16_bf16
//       on 4 independent accumulators from operands (bf16, >= 1024 elements, 16-byte aligned).
//       out: n_wg * 256 * waves_per_simd floats; stamps: 4 per wave.
//   fa_ceil_mix(operands, out, stamps, waves_per_simd, n_exp, n_fma, n_wg, iters, stream)
//       as fa_ceil_mfma, but each MFMA is followed by n_exp v_exp_f32 and n_fma v_fma_f32 (independent
//       of the MFMAs); (n_exp, n_fma) one of the pairs of FA_CEIL_MIXES.
//   fa_ceil_read_vgpr(src, bytes, out, stamps, n_wg, stream)
//       reads src[0, bytes) once with 16-byte loads into VGPRs (grid-stride, coalesced);
//       bytes a positive multiple of 16, src 16-byte aligned; out: 16 bytes (written only in the
//       practically impossible case that the XOR of everything read is a fixed pattern).
//   fa_ceil_read_lds(src, bytes, stamps, n_wg, stream)
//       reads src[0, bytes) once with buffer loads that write LDS directly, 64 KiB per workgroup
//       iteration (each wave 16 KiB, 16 loads of 1 KiB), two iterations in flight per wave;
//       bytes a positive multiple of 65536, src 16-byte aligned.
//   fa_ceil_lds(out, stamps, n_wg, iters, transpose, stream)
//       every wave reads 64 KiB of LDS iters times: 64 ds_read_b128 of 1 KiB (transpose = 0) or 128
//       ds_read_b64_tr_b16 of 512 bytes with the fused kernel's V-tile addressing (transpose = 1)
//       per pass, conflict-free; out: n_wg * 256 * 4 uint32.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "fa_device.h"

namespace {

using fa::bf16x8;
using fa::f32x16;
using fa::i16x4;
using fa::lds_i16x4;
using fa::u32x4;

__device__ __forceinline__ void stamp_begin(uint64_t& clk, uint64_t& real) {
  clk = __builtin_amdgcn_s_memtime();
  real = __builtin_amdgcn_s_memrealtime();
}
__device__ __forceinline__ void stamp_end(uint64_t* stamps, uint64_t clk0, uint64_t real0) {
  const uint64_t clk1 = __builtin_amdgcn_s_memtime();
  const uint64_t real1 = __builtin_amdgcn_s_memrealtime();
  const int wave = (blockIdx.x * blockDim.x + threadIdx.x) >> 6;
  if ((threadIdx.x & 63) == 0) {
    stamps[4 * wave + 0] = clk0;
    stamps[4 * wave + 1] = clk1;
    stamps[4 * wave + 2] = real0;
    stamps[4 * wave + 3] = real1;
  }
}

constexpr int kMfmaLds = 96 * 1024;  // holds a CU: one workgroup per CU

template <int WPE>
__global__ __attribute__((amdgpu_flat_work_group_size(256 * WPE, 256 * WPE), amdgpu_waves_per_eu(WPE, WPE)))
void ceil_mfma_kernel(const uint16_t* __restrict__ operands, float* __restrict__ out, uint64_t* __restrict__ stamps,
                      int iters) {
  __shared__ unsigned char hold[kMfmaLds];
  const int lane = threadIdx.x & 63;
  const bf16x8 a = *reinterpret_cast<const bf16x8*>(operands + lane * 8);
  const bf16x8 b = *reinterpret_cast<const bf16x8*>(operands + 512 + lane * 8);
  f32x16 c0{}, c1{}, c2{}, c3{};
  uint64_t clk0, real0;
  stamp_begin(clk0, real0);
  for (int i = 0; i < iters; ++i) {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      c0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c0, 0, 0, 0);
      c1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c1, 0, 0, 0);
      c2 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c2, 0, 0, 0);
      c3 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c3, 0, 0, 0);
    }
  }
  stamp_end(stamps, clk0, real0);
  float s = 0.f;
#pragma unroll
  for (int r = 0; r < 16; ++r) s += c0[r] + c1[r] + c2[r] + c3[r];
  // touch the LDS reservation so that it is kept (one byte per workgroup, written and read back)
  if (threadIdx.x == 0) hold[blockIdx.x % kMfmaLds] = (unsigned char)iters;
  __syncthreads();
  out[blockIdx.x * blockDim.x + threadIdx.x] = s + (float)hold[blockIdx.x % kMfmaLds];
}

// Issue cost of the online softmax's VALU work next to the MFMAs (the counterpart of the paper's
// instruction-count ceiling): every slot is one v_mfma_f32_32x32x16_bf16 (4 independent accumulators
// in turn) followed by NE v_exp_f32 and NF v_fma_f32 on 16 independent registers (each register is
// updated once per 4 slots when NE + NF = 4), issued in exactly this order. The stamps give the
// shader cycles per slot.
template <int WPE, int NE, int NF>
__global__ __attribute__((amdgpu_flat_work_group_size(256 * WPE, 256 * WPE), amdgpu_waves_per_eu(WPE, WPE)))
void ceil_mix_kernel(const uint16_t* __restrict__ operands, float* __restrict__ out, uint64_t* __restrict__ stamps,
                     int iters) {
  __shared__ unsigned char hold[kMfmaLds];
  const int lane = threadIdx.x & 63;
  const bf16x8 a = *reinterpret_cast<const bf16x8*>(operands + lane * 8);
  const bf16x8 b = *reinterpret_cast<const bf16x8*>(operands + 512 + lane * 8);
  f32x16 c[4] = {};
  float x[16];
#pragma unroll
  for (int k = 0; k < 16; ++k) x[k] = 0.0625f * (float)(k + 1) + 0.001f * (float)lane;
  uint64_t clk0, real0;
  stamp_begin(clk0, real0);
  // Volatile asm statements keep their order; no instruction reads a register another one wrote
  // within the same slot, so no wait states are needed.
  for (int i = 0; i < iters; ++i) {
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      asm volatile("v_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+v"(c[u]) : "v"(a), "v"(b));
#pragma unroll
      for (int e = 0; e < NE; ++e) asm volatile("v_exp_f32 %0, -|%0|" : "+v"(x[(u * (NE + NF) + e) & 15]));
#pragma unroll
      for (int f = 0; f < NF; ++f) asm volatile("v_fma_f32 %0, %0, 0.5, 0.5" : "+v"(x[(u * (NE + NF) + NE + f) & 15]));
    }
  }
  stamp_end(stamps, clk0, real0);
  float s = 0.f;
#pragma unroll
  for (int k = 0; k < 16; ++k) s += x[k];
#pragma unroll
  for (int u = 0; u < 4; ++u)
#pragma unroll
    for (int r = 0; r < 16; ++r) s += c[u][r];
  if (threadIdx.x == 0) hold[blockIdx.x % kMfmaLds] = (unsigned char)iters;
  __syncthreads();
  out[blockIdx.x * blockDim.x + threadIdx.x] = s + (float)hold[blockIdx.x % kMfmaLds];
}

__global__ __launch_bounds__(256) void ceil_read_vgpr_kernel(const u32x4* __restrict__ src, uint64_t n16,
                                                             u32x4* __restrict__ out, uint64_t* __restrict__ stamps) {
  uint64_t clk0, real0;
  stamp_begin(clk0, real0);
  const uint64_t stride = (uint64_t)gridDim.x * blockDim.x;
  uint64_t i = (uint64_t)blockIdx.x * blockDim.x + threadIdx.x;
  u32x4 acc = {0u, 0u, 0u, 0u};
  for (; i + 3 * stride < n16; i += 4 * stride) {
    const u32x4 x0 = src[i], x1 = src[i + stride], x2 = src[i + 2 * stride], x3 = src[i + 3 * stride];
    acc ^= x0 ^ x1 ^ x2 ^ x3;
  }
  for (; i < n16; i += stride) acc ^= src[i];
  stamp_end(stamps, clk0, real0);
  if (acc.x == 0x9e3779b9u && acc.y == 0x7f4a7c15u && acc.z == 0x85ebca6bu && acc.w == 0xc2b2ae35u) out[0] = acc;
}

constexpr int kLdsChunk = 65536;              // bytes per workgroup iteration
constexpr int kLdsWaveBytes = kLdsChunk / 4;  // 16 loads of 1 KiB per wave

__global__ __launch_bounds__(256) void ceil_read_lds_kernel(const unsigned char* __restrict__ src, int n_chunks,
                                                            uint64_t* __restrict__ stamps) {
  __shared__ __attribute__((aligned(1024))) unsigned char sink[4 * kLdsWaveBytes];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const uint32_t lds = fa::lds_offset(sink + wave * kLdsWaveBytes);
  uint64_t clk0, real0;
  stamp_begin(clk0, real0);
  for (int c = blockIdx.x; c < n_chunks; c += gridDim.x) {
    const uint64_t base = reinterpret_cast<uint64_t>(src) + (uint64_t)c * kLdsChunk + (uint64_t)wave * kLdsWaveBytes;
    const u32x4 rsrc = {(uint32_t)base, (uint32_t)(base >> 32) & 0xffffu, (uint32_t)kLdsWaveBytes, 0x00020000u};
#pragma unroll
    for (int k = 0; k < 16; ++k) fa::dma16_buffer(rsrc, (uint32_t)(k * 1024 + lane * 16), lds + k * 1024);
    fa::wait_vmcnt<16>();  // the previous iteration's 16 loads have landed; this one's stay in flight
  }
  fa::wait_vmcnt<0>();
  stamp_end(stamps, clk0, real0);
}

constexpr int kLdsBytes = 65536;

template <bool TR>
__global__ __launch_bounds__(256) void ceil_lds_kernel(uint32_t* __restrict__ out, uint64_t* __restrict__ stamps,
                                                      int iters) {
  __shared__ __attribute__((aligned(1024))) unsigned char buf[kLdsBytes];
  for (int i = threadIdx.x; i < kLdsBytes / 4; i += blockDim.x)
    reinterpret_cast<uint32_t*>(buf)[i] = (uint32_t)i * 2654435761u;
  __syncthreads();
  const int lane = threadIdx.x & 63;
  uint64_t clk0, real0;
  stamp_begin(clk0, real0);
  u32x4 acc = {0u, 0u, 0u, 0u};
  for (int it = 0; it < iters; ++it) {
    if constexpr (!TR) {
      // 64 reads of 1 KiB (64 lanes x 16 contiguous bytes: 16 different bank slots per 16 lanes)
#pragma unroll 16
      for (int u = 0; u < 64; ++u) {
        const int blk = (u + it) & 63;
        acc ^= *reinterpret_cast<const u32x4*>(buf + blk * 1024 + lane * 16);
      }
    } else {
      // 128 transpose reads of 512 bytes with the fused kernel's V-fragment addressing at d_v = 128
      // (four 64-key tiles of 256-byte rows, 16-byte chunks swizzled by key mod 4): tile, 16-key
      // step ps, 32-dim block db, and the second half 4 keys further on
      const int v_key = 8 * (lane >> 5) + ((lane & 15) >> 2);
      const int v_t = (2 * ((lane >> 4) & 1) + ((lane & 3) >> 1)) ^ fa::v_swizzle<128>(v_key);
      const int v_half = (lane & 1) * 8;
#pragma unroll 16
      for (int u = 0; u < 128; ++u) {
        const int tile = ((u >> 5) + it) & 3, ps = (u >> 3) & 3, db = (u >> 1) & 3, hi = u & 1;
        const int off = tile * 16384 + (ps * 16 + v_key + 4 * hi) * 256 + (((db * 4) ^ v_t) << 4) + v_half;
        const i16x4 x = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(buf + off));
        const auto w = fa::bit_cast<fa::f32x2>(x);
        acc.x ^= __float_as_uint(w.x);
        acc.y ^= __float_as_uint(w.y);
      }
    }
  }
  stamp_end(stamps, clk0, real0);
  reinterpret_cast<u32x4*>(out)[blockIdx.x * blockDim.x + threadIdx.x] = acc;
}

}  // namespace

extern "C" {

int fa_ceil_mfma(const void* operands, float* out, unsigned long long* stamps, int waves_per_simd, int n_wg, int iters,
                 hipStream_t stream) {
  if (operands == nullptr || out == nullptr || stamps == nullptr || n_wg <= 0 || iters <= 0 ||
      (reinterpret_cast<uintptr_t>(operands) & 15) != 0 || (waves_per_simd != 1 && waves_per_simd != 2))
    return hipErrorInvalidValue;
  const uint16_t* op = static_cast<const uint16_t*>(operands);
  uint64_t* st = reinterpret_cast<uint64_t*>(stamps);
  if (waves_per_simd == 1)
    hipLaunchKernelGGL(ceil_mfma_kernel<1>, dim3(n_wg), dim3(256), 0, stream, op, out, st, iters);
  else
    hipLaunchKernelGGL(ceil_mfma_kernel<2>, dim3(n_wg), dim3(512), 0, stream, op, out, st, iters);
  return hipGetLastError();
}

// Instruction mixes of fa_ceil_mix: (exponentials, fmas) per MFMA slot.
#define FA_CEIL_MIXES(X) X(0, 0) X(0, 2) X(0, 4) X(0, 6) X(0, 8) X(1, 0) X(2, 0) X(1, 2) X(1, 3) X(1, 4) X(2, 2) X(2, 4)

int fa_ceil_mix(const void* operands, float* out, unsigned long long* stamps, int waves_per_simd, int n_exp,
                int n_fma, int n_wg, int iters, hipStream_t stream) {
  if (operands == nullptr || out == nullptr || stamps == nullptr || n_wg <= 0 || iters <= 0 ||
      (reinterpret_cast<uintptr_t>(operands) & 15) != 0 || (waves_per_simd != 1 && waves_per_simd != 2))
    return hipErrorInvalidValue;
  const uint16_t* op = static_cast<const uint16_t*>(operands);
  uint64_t* st = reinterpret_cast<uint64_t*>(stamps);
#define FA_CEIL_MIX_CASE(E, F)                                                                          \
  if (n_exp == E && n_fma == F) {                                                                       \
    if (waves_per_simd == 1)                                                                            \
      hipLaunchKernelGGL((ceil_mix_kernel<1, E, F>), dim3(n_wg), dim3(256), 0, stream, op, out, st, iters); \
    else                                                                                                \
      hipLaunchKernelGGL((ceil_mix_kernel<2, E, F>), dim3(n_wg), dim3(512), 0, stream, op, out, st, iters); \
    return hipGetLastError();                                                                           \
  }
  FA_CEIL_MIXES(FA_CEIL_MIX_CASE)
#undef FA_CEIL_MIX_CASE
  return hipErrorInvalidValue;
}

int fa_ceil_read_vgpr(const void* src, size_t bytes, void* out, unsigned long long* stamps, int n_wg,
                      hipStream_t stream) {
  if (src == nullptr || out == nullptr || stamps == nullptr || n_wg <= 0 || bytes == 0 || bytes % 16 != 0 ||
      (reinterpret_cast<uintptr_t>(src) & 15) != 0)
    return hipErrorInvalidValue;
  hipLaunchKernelGGL(ceil_read_vgpr_kernel, dim3(n_wg), dim3(256), 0, stream, static_cast<const u32x4*>(src),
                     (uint64_t)(bytes / 16), static_cast<u32x4*>(out), reinterpret_cast<uint64_t*>(stamps));
  return hipGetLastError();
}

int fa_ceil_read_lds(const void* src, size_t bytes, unsigned long long* stamps, int n_wg, hipStream_t stream) {
  if (src == nullptr || stamps == nullptr || n_wg <= 0 || bytes == 0 || bytes % kLdsChunk != 0 ||
      bytes / kLdsChunk > (size_t)INT32_MAX || (reinterpret_cast<uintptr_t>(src) & 15) != 0)
    return hipErrorInvalidValue;
  hipLaunchKernelGGL(ceil_read_lds_kernel, dim3(n_wg), dim3(256), 0, stream, static_cast<const unsigned char*>(src),
                     (int)(bytes / kLdsChunk), reinterpret_cast<uint64_t*>(stamps));
  return hipGetLastError();
}

int fa_ceil_lds(void* out, unsigned long long* stamps, int n_wg, int iters, int transpose, hipStream_t stream) {
  if (out == nullptr || stamps == nullptr || n_wg <= 0 || iters <= 0) return hipErrorInvalidValue;
  uint32_t* o = static_cast<uint32_t*>(out);
  uint64_t* st = reinterpret_cast<uint64_t*>(stamps);
  if (transpose)
    hipLaunchKernelGGL(ceil_lds_kernel<true>, dim3(n_wg), dim3(256), 0, stream, o, st, iters);
  else
    hipLaunchKernelGGL(ceil_lds_kernel<false>, dim3(n_wg), dim3(256), 0, stream, o, st, iters);
  return hipGetLastError();
}

}  // extern "C"
