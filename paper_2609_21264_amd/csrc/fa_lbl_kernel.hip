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
//    the direct-to-LDS buffer loads of the fused kernel, two tiles ahead in a three-slot ring (one
//    tile ahead in two slots for d_qk = 192). With
//    the K rows in the permuted order perm32, each lane's accumulator holds 8 consecutive keys of
//    one query row per register group; the tile is staged through LDS so that every store writes
//    whole 128-byte row segments.
//  * softmax: one wavefront per row, 16-byte loads and stores (1 KiB contiguous per instruction).
//    A row of up to 8192 keys stays in registers between the statistics and the write; longer rows
//    are read twice.
//  * P V: one workgroup per block of 128 query rows computing O^T = V^T P^T; P and V tiles both go
//    HBM -> LDS by direct-to-LDS loads (P in whole 128-byte row segments) through a ring, and V is
//    read with ds_read_b64_tr_b16 as in the fused kernel.
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

// Buffer descriptor over [base, base + bytes): lanes whose access lies past the end read zeros and
// write nothing.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(base, (short)0, (int)bytes, 0x00020000);
}

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
  // K ring slots; tile j + NKR - 1 is loaded during step j. Two slots for the widest head keep the
  // workgroup's LDS at 64 KiB (two workgroups per CU).
  constexpr int NKR = DQK >= 192 ? 2 : 3;
  constexpr int D = NKR - 1;
  constexpr int KL = kLblKeys * KCH / 64 / kWaves;      // direct-to-LDS loads per wave per tile
  constexpr int NST = 4;                                // S stores per wave per tile
  static_assert(KL * 64 * kWaves == kLblKeys * KCH, "tile split over waves");
  static_assert(KL + 2 * NST < 64, "vmcnt range");
  constexpr int STAGE = 32 * kLblKeys * 2;              // one wave's 32 x 64 tile of S, bf16
  __shared__ __attribute__((aligned(1024))) unsigned char smem[NKR * K_BYTES + kWaves * STAGE];

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
  // The wave's tile goes through LDS so that each store writes 8 whole 128-byte row segments (lane l:
  // row 8 s + l / 8 of the wave, chunk l % 8); stored from the accumulator layout, every instruction
  // would write 32 rows 32 bytes at a time. Chunk c of tile row r sits at chunk c ^ ((r >> 1) & 7) of
  // the row: the 16 lanes the LDS serves per cycle then hit 16 different 16-byte bank slots when
  // writing (16 rows, one chunk) and when reading (2 rows, 8 chunks).
  unsigned char* stage = smem + NKR * K_BYTES + wave * STAGE;
  const int st_row = lane >> 3, st_c = lane & 7;
  const uint32_t out_off = (uint32_t)((wave * 32 + st_row) * p.ld + 8 * st_c) * 2u;

  // Per wave the vector-memory instructions go: K0 .. K(D-1), then per step j: K(j+D), S(j) (4
  // stores). Before step j, K(j) must have landed; issued after it are: for j >= D, S(j-D) and the
  // D - 1 steps after it (a K tile and 4 stores each); for j < D, K(j+1) .. K(D-1) and the j steps so
  // far. Vector memory operations complete in issue order for the counter.
  static_assert(D == 1 || D == 2, "prefetch distance");
#pragma unroll
  for (int t = 0; t < D; ++t) kload.issue(t * kLblKeys, kslot(t), wave);
  for (int j = 0; j < nt; ++j) {
    if (j >= D)
      fenced_wait<NST + (D - 1) * (KL + NST)>();
    else if (j == 1)
      fenced_wait<KL + NST>();  // D == 2
    else
      fenced_wait<(D - 1) * KL>();
    // The barrier publishes K(j) and ensures every wave is done with step j-1, whose slot K(j+D) reuses.
    block_barrier();
    kload.issue((j + D) * kLblKeys, kslot(j + D), wave);
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
    // Register 8*g + r of acc[kb] holds key j*64 + 32*kb + 16*g + 8*h + r of row rl (r < 8): chunk
    // 4*kb + 2*g + h of the tile row i32.
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int g = 0; g < 2; ++g) {
        u32x4 w;
#pragma unroll
        for (int t = 0; t < 4; ++t)
          w[t] = pack_bf16x2(acc[kb][8 * g + 2 * t] * p.scale, acc[kb][8 * g + 2 * t + 1] * p.scale);
        const int c = 4 * kb + 2 * g + h;
        *reinterpret_cast<u32x4*>(stage + i32 * 128 + ((c ^ ((i32 >> 1) & 7)) << 4)) = w;
      }
    const uint32_t tile_off = out_off + (uint32_t)(j * kLblKeys) * 2u;
#pragma unroll
    for (int st = 0; st < NST; ++st) {
      const int r = 8 * st + st_row;
      const u32x4 w = *reinterpret_cast<const u32x4*>(stage + r * 128 + ((st_c ^ ((r >> 1) & 7)) << 4));
      __builtin_amdgcn_raw_buffer_store_b128(w, out, (int)(tile_off + (uint32_t)(8 * st * p.ld) * 2u), 0, 0);
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

// One wavefront per row. The row's chunks (8 keys, 16 bytes) are held in registers in groups of
// 64 * NCH: lane l holds chunks g0 + 64 t + l. Masked keys are replaced by bf16 -inf as they are
// loaded, so the arithmetic below needs no mask: their exponentials are 0 and they never win a
// maximum. Chunks past the row are skipped with wave-uniform branches.
template <int NCH>
__global__ __launch_bounds__(256) void lbl_softmax_kernel(LblParams p) {
  constexpr float kLog2e = 1.44269504088896340736f;
  constexpr float kLn2 = 0.69314718055994530942f;
  constexpr uint32_t kNegInf2 = 0xff80ff80u;  // two bf16 -inf
  constexpr int GROUP = 64 * NCH;             // chunks per register-resident group of a row
  const int lane = threadIdx.x & 63;
  const int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  if (r >= p.rows) return;
  const int bh = p.bh0 + (int)(r / p.sq);
  const int i = p.qb0 * kLblRows + (int)(r % p.sq);
  const int nvis = p.causal ? max(0, min(p.sk, i + 1 + p.sk - p.sq)) : p.sk;
  const int nr = (nvis + 7) / 8;                    // chunks holding a visible key
  const int nw = lbl_extent(p, i / kLblRows) / 8;   // chunks written
  const u32x4* src = reinterpret_cast<const u32x4*>(p.s + r * p.ld);
  u32x4* dst = reinterpret_cast<u32x4*>(p.p + r * p.ld);

  // Chunks of the group at g0 that hold a visible key (wave-uniform count of the t's that do).
  auto group_steps = [&](int g0, int n) { return min(NCH, (max(n - g0, 0) + 63) / 64); };
  auto load_group = [&](u32x4 (&buf)[NCH], int g0) {
    const int nt = group_steps(g0, nr);
#pragma unroll
    for (int t = 0; t < NCH; ++t) {
      if (t < nt) {
        const int c = g0 + t * 64 + lane;
        u32x4 x = c < nr ? src[c] : u32x4{kNegInf2, kNegInf2, kNegInf2, kNegInf2};
        if (c == nr - 1 && (nvis & 7)) {  // the chunk with the last visible key: mask its tail
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            const int k0 = 2 * e - (nvis & 7);  // element 2e is visible iff k0 < 0
            const uint32_t lo = k0 < 0 ? (x[e] & 0xffffu) : 0xff80u;
            const uint32_t hi = k0 + 1 < 0 ? (x[e] & 0xffff0000u) : 0xff800000u;
            x[e] = lo | hi;
          }
        }
        buf[t] = x;
      }
    }
  };

  // Statistics in the log2 domain: per lane an online maximum m (of the raw scores) and sum
  // l = sum 2^((s - m) log2 e) over the groups, then across the wave.
  u32x4 buf[NCH];
  float m = -INFINITY, l = 0.f;
  for (int g0 = 0; g0 < nr; g0 += GROUP) {
    load_group(buf, g0);
    const int nt = group_steps(g0, nr);
    float gm = -INFINITY;
#pragma unroll
    for (int t = 0; t < NCH; ++t)
      if (t < nt)
#pragma unroll
        for (int e = 0; e < 8; ++e) gm = fmaxf(gm, chunk_elem(buf[t], e));
    const float mn = fmaxf(m, gm);
    if (mn != -INFINITY) {
      const float c = mn * kLog2e;
      float s = 0.f;
#pragma unroll
      for (int t = 0; t < NCH; ++t)
        if (t < nt)
#pragma unroll
          for (int e = 0; e < 8; ++e) s += __builtin_amdgcn_exp2f(fmaf(chunk_elem(buf[t], e), kLog2e, -c));
      l = (m == -INFINITY ? 0.f : l * __builtin_amdgcn_exp2f((m - mn) * kLog2e)) + s;
      m = mn;
    }
    // Keep only the raw chunks live between the passes (the widened values are recomputed).
#pragma unroll
    for (int t = 0; t < NCH; ++t) asm volatile("" : "+v"(buf[t]));
  }
  const float M = wave_max(m);
  const float L = wave_sum(m == -INFINITY ? 0.f : l * __builtin_amdgcn_exp2f((m - M) * kLog2e));
  // P = 2^(s log2 e - off) with off = M log2 e + log2 L; a row without a visible key gets off = +inf,
  // hence P = 0, and LSE = -inf.
  const bool empty = M == -INFINITY;
  const float off = empty ? INFINITY : fmaf(M, kLog2e, __builtin_amdgcn_logf(L));
  if (lane == 0 && p.lse != nullptr) p.lse[(int64_t)bh * p.sq + i] = empty ? -INFINITY : off * kLn2;

  for (int g0 = 0; g0 < nw; g0 += GROUP) {
    if (nr > GROUP) load_group(buf, g0);  // otherwise the row's visible chunks are still in buf
    const int nt_vis = group_steps(g0, nr), nt_w = group_steps(g0, nw);
#pragma unroll
    for (int t = 0; t < NCH; ++t) {
      if (t < nt_w) {
        const int c = g0 + t * 64 + lane;
        u32x4 w = {0u, 0u, 0u, 0u};
        if (t < nt_vis && c < nr) {
#pragma unroll
          for (int e = 0; e < 4; ++e)
            w[e] = pack_bf16x2(__builtin_amdgcn_exp2f(fmaf(chunk_elem(buf[t], 2 * e), kLog2e, -off)),
                               __builtin_amdgcn_exp2f(fmaf(chunk_elem(buf[t], 2 * e + 1), kLog2e, -off)));
        }
        if (c < nw) dst[c] = w;
      }
    }
  }
}

// ---- 3. P V ---------------------------------------------------------------------------------------

#ifndef FA_LBL_PV_SLOTS
#define FA_LBL_PV_SLOTS 2
#endif

template <int DV>
__global__ __launch_bounds__(kWaves * 64) void lbl_pv_kernel(LblParams p) {
  constexpr int DB = DV / 32;                           // 32-dim blocks of the output
  constexpr int VCH = DV / 8;                           // 16-byte chunks per V row
  constexpr int V_BYTES = kLblKeys * DV * 2;
  constexpr int P_BYTES = kLblRows * kLblKeys * 2;      // the block's 128 rows x 64 keys of P
  constexpr int NR = FA_LBL_PV_SLOTS;                   // ring slots (V and P tiles); NR - 1 tiles ahead
  constexpr int VL = kLblKeys * VCH / 64 / kWaves;      // direct-to-LDS loads per wave per V tile
  constexpr int PL = P_BYTES / 1024 / kWaves;           // ... per P tile
  constexpr int PS = kLblKeys / 16;                     // k-steps per tile
  static_assert(NR >= 2, "at least double buffering");
  static_assert(VL * 64 * kWaves == kLblKeys * VCH && PL * 1024 * kWaves == P_BYTES, "tile split over waves");
  static_assert((NR - 1) * (VL + PL) < 64, "vmcnt range");
  __shared__ __attribute__((aligned(1024))) unsigned char smem[NR * (V_BYTES + P_BYTES)];

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
  auto vslot = [&](int t) { return smem + (t % NR) * V_BYTES; };
  auto pslot = [&](int t) { return smem + NR * V_BYTES + (t % NR) * P_BYTES; };
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

  // P tiles (128 rows x 64 keys, 128-byte rows in LDS) arrive by direct-to-LDS loads, 8 whole row
  // segments per instruction. Chunk c of tile row r sits at chunk c ^ ((r >> 1) & 7), which keeps
  // both the loads and the B-operand reads (16 rows, one chunk per 16 lanes) free of bank conflicts;
  // the swizzle is in each lane's source offset. Each tile is a buffer starting at its first key,
  // ending with the block's last row; padding rows and tiles past the extent (empty buffer) load
  // zeros without a memory access.
  const uint64_t p_base = reinterpret_cast<uint64_t>(p.p + lbl_chunk_row(p, bh, qb) * p.ld);
  const uint32_t p_bytes = (uint32_t)(rows_here * p.ld * 2);
  uint32_t p_voff[PL];
#pragma unroll
  for (int i = 0; i < PL; ++i) {
    const int pch = (wave * PL + i) * 64 + lane;  // physical 16-byte chunk of the tile
    const int r = pch >> 3, c = (pch & 7) ^ ((r >> 1) & 7);
    p_voff[i] = (uint32_t)(r * p.ld + 8 * c) * 2u;
  }
  auto issue = [&](int t) {
    vload.issue(t * kLblKeys, vslot(t), wave);
    const uint32_t key_bytes = (uint32_t)(t * kLblKeys) * 2u;
    const uint64_t base = p_base + key_bytes;
    const u32x4 rs = {(uint32_t)base, (uint32_t)(base >> 32) & 0xffffu, t < nt ? p_bytes - key_bytes : 0u,
                      0x00020000u};
    const uint32_t l = lds_offset(pslot(t) + wave * PL * 1024);
#pragma unroll
    for (int i = 0; i < PL; ++i) dma16_buffer(rs, p_voff[i], l + i * 1024);
  };
  // B operand P^T[keys 16*ps + 0..15][rows of the wave]: lane (i32, h) reads row rl, chunk 2*ps + h.
  auto pfrag = [&](const unsigned char* sP, int ps) {
    const int c = (2 * ps + h) ^ ((rl >> 1) & 7);
    return *reinterpret_cast<const bf16x8*>(sP + rl * 128 + (c << 4));
  };

  f32x16 oacc[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) oacc[db] = f32x16{};

  // Per wave the loads go V0 P0 V1 P1 .. (prologue, NR - 1 tiles), then per step j: V(j+NR-1)
  // P(j+NR-1). Before step j, tile j must have landed; issued after it are the NR - 2 tiles after it.
#pragma unroll
  for (int t = 0; t < NR - 1; ++t) issue(t);
  for (int j = 0; j < nt; ++j) {
    fenced_wait<(NR - 2) * (VL + PL)>();
    block_barrier();  // publishes tile j; every wave is done with tile j-1, whose slot the next load reuses
    issue(j + NR - 1);
    const unsigned char* sV = vslot(j);
    const unsigned char* sP = pslot(j);
#pragma unroll
    for (int ps = 0; ps < PS; ++ps) {
      const bf16x8 pf = pfrag(sP, ps);
#pragma unroll
      for (int db = 0; db < DB; ++db)
        oacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vfrag(sV, ps, db), pf, oacc[db], 0, 0, 0);
    }
  }
  // No direct-to-LDS load may still be in flight when the workgroup exits.
  fenced_wait<0>();

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
