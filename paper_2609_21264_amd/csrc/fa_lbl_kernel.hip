// Layer-by-layer (unfused) attention forward for gfx950: the paper's diagnostic baseline mapping
// (Sec. "Diagnostic Baseline: Unfused Layer-by-Layer Attention") as three kernels that run one after
// another, each reading its input from HBM and writing its result back, with the score matrix and the
// probability matrix spilled in bf16 (Table 3):
//
//   1. lbl_scores_kernel:  S = bf16(scale * Q K^T)                  bf16 MFMA, fp32 accumulation
//   2. lbl_softmax_kernel: LSE_i = ln sum_{j visible} exp(S_ij);
//                          P_ij = bf16(exp(S_ij - LSE_i)) on visible keys, 0 on masked ones
//   3. lbl_pv_kernel:      O = bf16(P V)                            bf16 MFMA, fp32 accumulation
//
// Per score element the spill costs 2 bytes written and read for S and again for P, against
// 2 * (d_qk + d_v) flops: the whole path's intensity is below d / 2 flop per byte (Sec. "The
// Operational Intensity Constraint", Table 3), under MI355X's ridge point for any head dimension
// here, so every kernel is written to stream HBM:
//  * scores: one workgroup per block of 128 query rows. The block's Q rows stay in registers as the
//    B operand of S^T = K Q^T (v_mfma_f32_32x32x16_bf16); 64-key K tiles go HBM/L2 -> LDS through
//    the direct-to-LDS buffer loads of the fused kernel, two tiles ahead in a three-slot ring. With
//    the K rows in the permuted order perm32, each lane's accumulator holds 8 consecutive keys of
//    one query row per register group, so every store writes 16 bytes of a row.
//  * softmax: one wavefront per row, 16-byte loads and stores (1 KiB contiguous per instruction).
//    A row of up to 8192 keys stays in registers between the statistics and the write; longer rows
//    are read twice.
//  * P V: one workgroup per block of 128 query rows; each lane loads its 16-byte fragments of P
//    straight into the B operand registers of O^T = V^T P^T, two tiles ahead; V tiles go through an
//    LDS ring and are read with ds_read_b64_tr_b16 as in the fused kernel.
//  * Causal masking: no kernel touches keys past a block's extent (the visible keys of its last row,
//    rounded up to 64); the softmax writes the masked entries inside the extent as zeros, so the
//    P V product needs no mask. Block order and XCD placement follow the fused kernel (heaviest
//    blocks first, the query heads of one key/value head on one XCD).
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "fa_device.h"
#include "fa_internal.h"

namespace fa {
namespace {

constexpr int kWaves = 4;  // wavefronts per workgroup of the scores and P V kernels (32 query rows each)
static_assert(kWaves * 32 == kLblRows, "one 32-row MFMA block per wave");

// Keys the rows of query block qb use: the visible keys of the block's last row, rounded up to whole
// key tiles.
__device__ __forceinline__ int lbl_extent(const LblParams& p, int qb) {
  int n = p.sk;
  if (p.causal) {
    const int last = min(p.sq, (qb + 1) * kLblRows) - 1;
    n = max(0, min(p.sk, last + 1 + p.sk - p.sq));
  }
  return (n + kLblKeys - 1) / kLblKeys * kLblKeys;
}

// First chunk row of unit (bh, qb).
__device__ __forceinline__ int64_t lbl_chunk_row(const LblParams& p, int bh, int qb) {
  return (int64_t)(bh - p.bh0) * p.sq + (int64_t)(qb - p.qb0) * kLblRows;
}

// Workgroup t -> unit (bh, qb). Workgroup t runs on XCD t % 8; units are ordered heaviest query block
// first (causal), then by group of xgroup query heads that share a key/value head, and each such
// group of units goes to one XCD, groups round-robin (the same placement as the fused kernel).
__device__ __forceinline__ void lbl_decode(int t, const LblParams& p, int& bh, int& qb) {
  const int G = p.xgroup;
  const int n = p.nbh * p.nqb;
  const int span = kNumXcd * G;
  const int full = (n / span) * span;
  int L = t;
  if (t < full) {
    const int xcd = t % kNumXcd, slot = t / kNumXcd;
    L = ((slot / G) * kNumXcd + xcd) * G + slot % G;
  }
  const int member = L % G;
  const int r = L / G;
  const int ngroups = p.nbh / G;
  const int qr = r / ngroups;
  qb = p.causal ? p.qb0 + p.nqb - 1 - qr : p.qb0 + qr;
  bh = p.bh0 + (r % ngroups) * G + member;
}

// Raw buffer descriptor over [base, base + bytes): lanes whose access lies past the end read zeros
// and write nothing.
__device__ __forceinline__ u32x4 raw_rsrc(const void* base, uint32_t bytes) {
  const uint64_t b = reinterpret_cast<uint64_t>(base);
  return u32x4{(uint32_t)b, (uint32_t)(b >> 32) & 0xffffu, bytes, 0x00020000u};
}
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(base, (short)0, (int)bytes, 0x00020000);
}

// 16 bytes of the buffer at byte voff into a VGPR quad, not tracked by the compiler (like the
// direct-to-LDS loads): the caller orders it with wait_vmcnt and then vgpr_ready(), which keeps
// every read of the registers after that wait.
__device__ __forceinline__ void load16_buffer(bf16x8& r, u32x4 rsrc, uint32_t voff) {
  asm volatile("buffer_load_dwordx4 %0, %1, %2, 0 offen" : "=v"(r) : "v"(voff), "s"(rsrc) : "memory");
}
__device__ __forceinline__ void vgpr_ready(bf16x8& r) { asm volatile("" : "+v"(r)); }

template <int N>
__device__ __forceinline__ void fenced_wait() {
  compiler_fence();
  wait_vmcnt<N>();
  compiler_fence();
}
__device__ __forceinline__ void block_barrier() {
  compiler_fence();
  __builtin_amdgcn_s_barrier();
  compiler_fence();
}

// ---- 1. scores ------------------------------------------------------------------------------------

template <int DQK>
__global__ __launch_bounds__(kWaves * 64) void lbl_scores_kernel(LblParams p) {
  constexpr int KS = DQK / 16;                          // k-steps of the product
  constexpr int KCH = DQK / 8;                          // 16-byte chunks per K row
  constexpr int K_BYTES = kLblKeys * DQK * 2;
  constexpr int NKR = 3;                                // K ring slots
  constexpr int KL = kLblKeys * KCH / 64 / kWaves;      // direct-to-LDS loads per wave per tile
  constexpr int NST = 4;                                // S stores per wave per tile
  static_assert(KL * 64 * kWaves == kLblKeys * KCH, "tile split over waves");
  static_assert(KL + 2 * NST < 64, "vmcnt range");
  __shared__ __attribute__((aligned(1024))) unsigned char smem[NKR * K_BYTES];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int i32 = lane & 31, h = lane >> 5;
  int bh, qb;
  lbl_decode(blockIdx.x, p, bh, qb);
  const int64_t kvh = (int64_t)(bh / p.hq) * p.hkv + (bh % p.hq) / p.group;
  const int nt = lbl_extent(p, qb) / kLblKeys;
  const int rows_here = min(kLblRows, p.sq - qb * kLblRows);
  const int rl = wave * 32 + i32;  // this lane's query row in the block

  // Q rows as B operands: lane (i32, h) holds row rl, dims 16*ks + 8*h .. +7. Padding rows of the last
  // block read the block's last row; their stores fall outside the output buffer.
  bf16x8 qf[KS];
  const uint16_t* qrow = p.q + ((int64_t)bh * p.sq + qb * kLblRows + min(rl, rows_here - 1)) * DQK + 8 * h;
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) qf[ks] = *reinterpret_cast<const bf16x8*>(qrow + 16 * ks);

  TileLoader<kWaves, kLblKeys, KCH> kload;
  kload.init(p.k + kvh * p.sk * DQK, min(p.sk, nt * kLblKeys), wave, lane, [](int r) { return k_swizzle<DQK>(r); });
  auto kslot = [&](int t) { return smem + (t % NKR) * K_BYTES; };

  const __amdgpu_buffer_rsrc_t out = make_rsrc(p.s + lbl_chunk_row(p, bh, qb) * p.ld, (uint32_t)(rows_here * p.ld * 2));
  const uint32_t out_off = (uint32_t)(rl * p.ld + 8 * h) * 2u;

  // Per wave the vector-memory instructions go: K0, K1, then per step j: K(j+2), S(j) (4 stores).
  // Before step j, K(j) must have landed; issued after it are K(j+1) (j = 0), K(j+1) and S(j-1)
  // (j = 1), S(j-2), K(j+1) and S(j-1) (j >= 2). Vector memory operations complete in issue order
  // for the counter.
  kload.issue(0, kslot(0), wave);
  kload.issue(kLblKeys, kslot(1), wave);
  for (int j = 0; j < nt; ++j) {
    if (j >= 2)
      fenced_wait<KL + 2 * NST>();
    else if (j == 1)
      fenced_wait<KL + NST>();
    else
      fenced_wait<KL>();
    // The barrier publishes K(j) and ensures every wave is done with step j-1, whose slot K(j+2) reuses.
    block_barrier();
    kload.issue((j + 2) * kLblKeys, kslot(j + 2), wave);
    const unsigned char* sK = kslot(j);
    f32x16 acc[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb) {
      const unsigned char* krow = sK + (kb * 32 + perm32(i32)) * (DQK * 2);
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        const u32x4 a = *reinterpret_cast<const u32x4*>(krow + (((2 * ks + h) ^ k_lane_swizzle<DQK>(i32)) << 4));
        acc[kb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bit_cast<bf16x8>(a), qf[ks], ks == 0 ? f32x16{} : acc[kb],
                                                           0, 0, 0);
      }
    }
    // Register 8*g + r of acc[kb] holds key j*64 + 32*kb + 16*g + 8*h + r of row rl (r < 8).
    const uint32_t tile_off = out_off + (uint32_t)(j * kLblKeys) * 2u;
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int g = 0; g < 2; ++g) {
        u32x4 w;
#pragma unroll
        for (int t = 0; t < 4; ++t)
          w[t] = pack_bf16x2(acc[kb][8 * g + 2 * t] * p.scale, acc[kb][8 * g + 2 * t + 1] * p.scale);
        __builtin_amdgcn_raw_buffer_store_b128(w, out, (int)(tile_off + (32 * kb + 16 * g) * 2), 0, 0);
      }
  }
  // No direct-to-LDS load may still be in flight when the workgroup exits.
  fenced_wait<0>();
}

// ---- 2. mask + softmax ------------------------------------------------------------------------------

__device__ __forceinline__ float wave_max(float x) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x = fmaxf(x, __shfl_xor(x, o));
  return x;
}
__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) x += __shfl_xor(x, o);
  return x;
}

// Element e (0..7) of a 16-byte chunk of bf16, widened to fp32 (exact).
__device__ __forceinline__ float chunk_elem(const u32x4& c, int e) {
  const uint32_t w = c[e >> 1];
  return __uint_as_float((e & 1) ? (w & 0xffff0000u) : (w << 16));
}

template <int NCH>
__global__ __launch_bounds__(256) void lbl_softmax_kernel(LblParams p) {
  constexpr float kLog2e = 1.44269504088896340736f;
  constexpr float kLn2 = 0.69314718055994530942f;
  constexpr int GROUP = 64 * NCH;  // 16-byte chunks per register-resident group of a row
  const int lane = threadIdx.x & 63;
  const int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (r >= p.rows) return;
  const int bh = p.bh0 + (int)(r / p.sq);
  const int i = p.qb0 * kLblRows + (int)(r % p.sq);
  const int nvis = p.causal ? max(0, min(p.sk, i + 1 + p.sk - p.sq)) : p.sk;
  const int nr = (nvis + 7) / 8;                          // chunks holding a visible key
  const int nw = lbl_extent(p, i / kLblRows) / 8;         // chunks written
  const u32x4* src = reinterpret_cast<const u32x4*>(p.s + r * p.ld);
  u32x4* dst = reinterpret_cast<u32x4*>(p.p + r * p.ld);

  auto load_group = [&](u32x4 (&buf)[NCH], int g0) {
#pragma unroll
    for (int t = 0; t < NCH; ++t) {
      const int c = g0 + t * 64 + lane;
      buf[t] = c < nr ? src[c] : u32x4{0u, 0u, 0u, 0u};
    }
  };
  // log2-domain score of element e of chunk t of the group at g0, -inf when masked
  auto score = [&](const u32x4 (&buf)[NCH], int g0, int t, int e) {
    const int key = (g0 + t * 64 + lane) * 8 + e;
    return key < nvis ? chunk_elem(buf[t], e) * kLog2e : -INFINITY;
  };

  // Statistics: per lane an online maximum and sum over the groups, then across the wave.
  u32x4 buf[NCH];
  float m = -INFINITY, l = 0.f;
  for (int g0 = 0; g0 < nr; g0 += GROUP) {
    load_group(buf, g0);
    float gm = -INFINITY;
#pragma unroll
    for (int t = 0; t < NCH; ++t)
#pragma unroll
      for (int e = 0; e < 8; ++e) gm = fmaxf(gm, score(buf, g0, t, e));
    const float mn = fmaxf(m, gm);
    if (mn != -INFINITY) {
      float s = 0.f;
#pragma unroll
      for (int t = 0; t < NCH; ++t)
#pragma unroll
        for (int e = 0; e < 8; ++e) s += __builtin_amdgcn_exp2f(score(buf, g0, t, e) - mn);
      l = (m == -INFINITY ? 0.f : l * __builtin_amdgcn_exp2f(m - mn)) + s;
      m = mn;
    }
  }
  const float M = wave_max(m);
  const float L = wave_sum(m == -INFINITY ? 0.f : l * __builtin_amdgcn_exp2f(m - M));
  // P = 2^(t - off) with off = M + log2 L (log2 of the row sum); a row without a visible key gets
  // off = +inf, hence P = 0, and LSE = -inf.
  const bool empty = M == -INFINITY;
  const float off = empty ? INFINITY : M + __builtin_amdgcn_logf(L);
  if (lane == 0 && p.lse != nullptr) p.lse[(int64_t)bh * p.sq + i] = empty ? -INFINITY : off * kLn2;

  for (int g0 = 0; g0 < nw; g0 += GROUP) {
    if (nr > GROUP) load_group(buf, g0);  // otherwise the whole row is still in buf (g0 == 0)
#pragma unroll
    for (int t = 0; t < NCH; ++t) {
      const int c = g0 + t * 64 + lane;
      if (c < nw) {
        u32x4 w;
#pragma unroll
        for (int e = 0; e < 4; ++e)
          w[e] = pack_bf16x2(__builtin_amdgcn_exp2f(score(buf, g0, t, 2 * e) - off),
                             __builtin_amdgcn_exp2f(score(buf, g0, t, 2 * e + 1) - off));
        dst[c] = w;
      }
    }
  }
}

// ---- 3. P V ---------------------------------------------------------------------------------------

template <int DV>
__global__ __launch_bounds__(kWaves * 64) void lbl_pv_kernel(LblParams p) {
  constexpr int DB = DV / 32;                           // 32-dim blocks of the output
  constexpr int VCH = DV / 8;                           // 16-byte chunks per V row
  constexpr int V_BYTES = kLblKeys * DV * 2;
  constexpr int NVR = 3;                                // V ring slots
  constexpr int VL = kLblKeys * VCH / 64 / kWaves;      // direct-to-LDS loads per wave per tile
  constexpr int PS = kLblKeys / 16;                     // k-steps per tile = P loads per lane per tile
  static_assert(VL * 64 * kWaves == kLblKeys * VCH, "tile split over waves");
  static_assert(2 * (VL + PS) < 64, "vmcnt range");
  __shared__ __attribute__((aligned(1024))) unsigned char smem[NVR * V_BYTES];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int i32 = lane & 31, h = lane >> 5;
  int bh, qb;
  lbl_decode(blockIdx.x, p, bh, qb);
  const int64_t kvh = (int64_t)(bh / p.hq) * p.hkv + (bh % p.hq) / p.group;
  const int nt = lbl_extent(p, qb) / kLblKeys;
  const int rows_here = min(kLblRows, p.sq - qb * kLblRows);
  const int rl = wave * 32 + i32;

  TileLoader<kWaves, kLblKeys, VCH> vload;
  vload.init(p.v + kvh * p.sk * DV, min(p.sk, nt * kLblKeys), wave, lane, [](int r) { return v_swizzle<DV>(r); });
  auto vslot = [&](int t) { return smem + (t % NVR) * V_BYTES; };
  // Lane constants of the V transpose read (group G = lane / 16, slot j = lane % 16): see vfrag.
  const int v_key = 8 * (lane >> 5) + ((lane & 15) >> 2);
  const int v_t = (2 * ((lane >> 4) & 1) + ((lane & 3) >> 1)) ^ v_swizzle<DV>(v_key);
  const int v_half = (lane & 1) * 8;
  // A operand V^T[dims 32*db + 0..31][keys 16*ps + 0..15] of the tile in sV.
  auto vfrag = [&](const unsigned char* sV, int ps, int db) {
    const unsigned char* base = sV + (ps * 16 + v_key) * (DV * 2) + (((db * 4) ^ v_t) << 4) + v_half;
    const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(base));
    const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(base + 4 * DV * 2));
    return bit_cast<bf16x8>(__builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
  };

  // P fragments (B operands): lane (i32, h) loads row rl, keys 64*t + 16*ps + 8*h .. +7. Padding rows
  // and tiles past the extent lie outside the buffer and read zeros without a memory access.
  const u32x4 prs = raw_rsrc(p.p + lbl_chunk_row(p, bh, qb) * p.ld, (uint32_t)(rows_here * p.ld * 2));
  const uint32_t p_off = (uint32_t)(rl * p.ld + 8 * h) * 2u;
  bf16x8 pf[3][PS];
  auto issue = [&](bf16x8 (&f)[PS], int t) {
    vload.issue(t * kLblKeys, vslot(t), wave);
    const uint32_t base = t < nt ? p_off + (uint32_t)(t * kLblKeys) * 2u : 0x80000000u;
#pragma unroll
    for (int ps = 0; ps < PS; ++ps) load16_buffer(f[ps], prs, base + 32u * ps);
  };

  f32x16 oacc[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) oacc[db] = f32x16{};

  // Per wave: V0 P0 V1 P1, then per step j: V(j+2) P(j+2). Before step j, P(j) (issued after V(j))
  // must have landed; issued after it are V(j+1) and P(j+1).
  issue(pf[0], 0);
  issue(pf[1], 1);
  auto step = [&](int j, bf16x8 (&cur)[PS], bf16x8 (&ahead)[PS]) {
    fenced_wait<VL + PS>();
    block_barrier();  // publishes V(j); every wave is done with V(j-1), whose slot V(j+2) reuses
    issue(ahead, j + 2);
#pragma unroll
    for (int ps = 0; ps < PS; ++ps) vgpr_ready(cur[ps]);
    const unsigned char* sV = vslot(j);
#pragma unroll
    for (int ps = 0; ps < PS; ++ps)
#pragma unroll
      for (int db = 0; db < DB; ++db)
        oacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vfrag(sV, ps, db), cur[ps], oacc[db], 0, 0, 0);
  };
  // P registers rotate over three sets: step j reads set j % 3 and refills set (j + 2) % 3.
  int j = 0;
  for (; j + 2 < nt; j += 3) {
    step(j, pf[0], pf[2]);
    step(j + 1, pf[1], pf[0]);
    step(j + 2, pf[2], pf[1]);
  }
  if (j < nt) {
    step(j, pf[0], pf[2]);
    if (j + 1 < nt) step(j + 1, pf[1], pf[0]);
  }
  // The last two steps' loads (past the extent, zeros) are never consumed by a step: they land after
  // this wait, and the registers of every set stay reserved for them until here.
  fenced_wait<0>();
#pragma unroll
  for (int s = 0; s < 3; ++s)
#pragma unroll
    for (int ps = 0; ps < PS; ++ps) vgpr_ready(pf[s][ps]);

  // O^T accumulator: register 4*g + c of oacc[db] holds dim 32*db + 8*g + 4*h + c of row rl.
  if (rl < rows_here) {
    uint16_t* orow = p.o + ((int64_t)bh * p.sq + qb * kLblRows + rl) * DV + 4 * h;
#pragma unroll
    for (int db = 0; db < DB; ++db)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const uint32_t lo = pack_bf16x2(oacc[db][4 * g], oacc[db][4 * g + 1]);
        const uint32_t hi = pack_bf16x2(oacc[db][4 * g + 2], oacc[db][4 * g + 3]);
        *reinterpret_cast<uint2*>(orow + 32 * db + 8 * g) = make_uint2(lo, hi);
      }
  }
}

}  // namespace

bool lbl_scores_supported(int d_qk) { return d_qk == 64 || d_qk == 128 || d_qk == 192; }
bool lbl_pv_supported(int d_v) { return d_v == 64 || d_v == 128; }

hipError_t launch_lbl_scores(const LblParams& p, int d_qk, hipStream_t stream) {
  const dim3 grid(p.nbh * p.nqb), block(kWaves * 64);
  switch (d_qk) {
    case 64: hipLaunchKernelGGL(lbl_scores_kernel<64>, grid, block, 0, stream, p); break;
    case 128: hipLaunchKernelGGL(lbl_scores_kernel<128>, grid, block, 0, stream, p); break;
    case 192: hipLaunchKernelGGL(lbl_scores_kernel<192>, grid, block, 0, stream, p); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_lbl_softmax(const LblParams& p, hipStream_t stream) {
  hipLaunchKernelGGL(lbl_softmax_kernel<16>, dim3((unsigned)((p.rows + 3) / 4)), dim3(256), 0, stream, p);
  return hipGetLastError();
}

hipError_t launch_lbl_pv(const LblParams& p, int d_v, hipStream_t stream) {
  const dim3 grid(p.nbh * p.nqb), block(kWaves * 64);
  switch (d_v) {
    case 64: hipLaunchKernelGGL(lbl_pv_kernel<64>, grid, block, 0, stream, p); break;
    case 128: hipLaunchKernelGGL(lbl_pv_kernel<128>, grid, block, 0, stream, p); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

}  // namespace fa
