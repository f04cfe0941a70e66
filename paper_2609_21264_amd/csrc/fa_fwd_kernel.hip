// Fused attention forward for gfx950 (MI355X): one kernel computes, per (batch, query head, block of
// query rows), O = softmax(scale * Q K^T) V with the online softmax of the paper's per-tile algorithm
// (Alg. 1, Sec. 2.1): key/value rows are streamed in tiles, each query row keeps a running maximum
// and a running sum, and the unnormalised output accumulator is rescaled when the maximum grows.
// Scores and probabilities live only in registers; K and V tiles are staged in LDS.
//
// Mapping onto CDNA4:
//  * A workgroup has NWAVES wavefronts of 64 lanes; each wave owns 32*QB query rows.
//  * Scores are computed transposed, S^T = K Q^T, with v_mfma_f32_32x32x16_bf16: the K tile (LDS)
//    is the A operand and the wave's Q rows (AGPRs, loaded once) are the B operand. In the 32x32
//    accumulator a lane then holds ONE query row (column = lane % 32) and 16 keys, so the row
//    maximum and row sum need only in-lane reductions plus one exchange between the two lane halves
//    (v_permlane32_swap).
//  * The A-operand rows of K are loaded in a permuted key order (bits 2 and 3 of the row index
//    swapped), which makes each 8-register group of the accumulator hold 8 consecutive keys. After
//    rounding to bf16, those registers are already the B operand of the second product
//    O^T += V^T P^T, so P never moves between lanes or through LDS.
//  * V^T is the A operand of that product and needs keys contiguous per lane. V tiles stay
//    row-major in LDS and are read with ds_read_b64_tr_b16: within each 16-lane group the
//    instruction gathers a 4 (keys) x 16 (dims) block and hands lane i the 4 keys of dim i.
//  * K/V tiles move HBM -> LDS with direct-to-LDS loads (global_load_lds_dwordx4): no VGPR staging
//    and no LDS write instructions. A ring of NS stages keeps NS-1 tiles in flight; one wait on this
//    wave's own loads plus one barrier per tile publishes a stage and frees the previous one.
//  * 16-byte LDS chunks are XOR-swizzled per row (K: by the reading lane's key slot; V: by
//    2*(key mod 4)) so that the lanes served together hit different banks. The swizzle is produced
//    by choosing each lane's global source address, since the load writes LDS lane-linearly.
//  * The output accumulators O and the Q operand live in AGPRs for the whole kernel (inline-asm
//    MFMAs with fixed register classes); scores, probabilities and LDS fragments use VGPRs.
//  * Causal masking skips key tiles above the diagonal entirely and applies the element mask only on
//    diagonal and tail tiles.
//  * Workgroup order: heaviest query blocks first when causal, and the Hq/Hkv query heads that share
//    a key/value head are dispatched consecutively onto the same XCD (workgroup IDs are assigned to
//    the 8 XCDs round-robin), so their K/V tiles are served from one L2.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "fa_internal.h"

namespace fa {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef short i16x8 __attribute__((ext_vector_type(8)));
typedef __attribute__((address_space(3))) i16x4 lds_i16x4;
typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(1))) const void global_cvoid;

#ifndef FA_SPREAD
#define FA_SPREAD 0
#endif
#ifndef FA_ORDER
#define FA_ORDER 1
#endif
#ifndef FA_SCORE_BUILTIN
#define FA_SCORE_BUILTIN 1
#endif

constexpr float kLn2 = 0.69314718055994530942f;
constexpr float kRescaleSlack = 8.0f;
constexpr float kOverflowSum = 256.0f;  // 2^kRescaleSlack
constexpr int kNumXcd = 8;

// Row order of a 32-key block in the score product's A operand: A-row i holds key perm32(i).
// With the 32x32 accumulator layout (register r of a lane in half h holds A-row
// 8*(r/4) + 4*h + r%4), register r then holds key 16*(r/8) + 8*h + r%8.
__device__ __forceinline__ int perm32(int i) { return (i & ~12) | ((i & 4) << 1) | ((i & 8) >> 1); }

// XOR swizzle of the 16-byte chunks of K-tile row `row`. The reading lanes 0..7 of a phase load
// rows perm32(0..7) (+32*kb), whose swizzles are 0..7.
__device__ __forceinline__ int k_swizzle(int row) { return perm32(row & 31) & 7; }

// XOR swizzle of the 16-byte chunks of V-tile row `key`: the four key rows a 16-lane group of the
// transpose read touches at once land in different 32-byte bank slots.
__device__ __forceinline__ int v_swizzle(int key) { return 2 * (key & 3); }

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

// Both products are issued through inline asm so that the register classes are fixed: the score
// accumulators S live in VGPRs (the softmax reads them), the output accumulators O and the Q operand
// live in AGPRs for the whole kernel. The compiler does not model hazards of inline asm, so:
//  * each asm MFMA starts with s_nop 1: a VGPR operand may have just been written by VALU (P by
//    v_cvt_pk_bf16_f32), which needs 2 wait states before an MFMA reads it;
//  * agpr_fence() / vgpr_fence() separate asm MFMA writes of an accumulator from compiler-generated
//    accesses (initialisation, rescale, epilogue, softmax) in both directions: 18 wait states cover
//    the 8-pass MFMA write-to-read distance, and the operand ties keep the order;
//  * consecutive MFMAs accumulating into exactly the same registers need no wait states (the
//    accumulator is forwarded).
__device__ __forceinline__ void mfma_score_first(f32x16& acc, const bf16x8& k, const bf16x8& q) {
  asm("s_nop 1\n\tv_mfma_f32_32x32x16_bf16 %0, %1, %2, 0" : "=&v"(acc) : "v"(k), "a"(q));
}
__device__ __forceinline__ void mfma_score(f32x16& acc, const bf16x8& k, const bf16x8& q) {
  asm("s_nop 1\n\tv_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+v"(acc) : "v"(k), "a"(q));
}
__device__ __forceinline__ void mfma_out(f32x16& acc, const bf16x8& v, const bf16x8& pt) {
  asm("s_nop 1\n\tv_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+a"(acc) : "v"(v), "v"(pt));
}
__device__ __forceinline__ void agpr_fence(f32x16& acc) {
  asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 3" : "+a"(acc));
}
__device__ __forceinline__ void vgpr_fence(f32x16& acc) {
  asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 3" : "+v"(acc));
}
// 16 bytes of Q straight into an AGPR tuple (only ever read by asm MFMAs, so it never needs a VGPR
// copy). Waits for the load before returning.
__device__ __forceinline__ bf16x8 load_q(const void* ptr) {
  bf16x8 r;
  asm volatile("global_load_dwordx4 %0, %1, off\n\ts_waitcnt vmcnt(0)" : "=a"(r) : "v"(ptr) : "memory");
  return r;
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

template <int DQK_, int DV_, int BN_, int NWAVES_, int QB_, int WPE_, int NS_, int PIPE_, bool CAUSAL_>
struct Cfg {
  static constexpr int DQK = DQK_, DV = DV_, BN = BN_, NWAVES = NWAVES_, QB = QB_, WPE = WPE_, NS = NS_;
  // 0: one tile per step; 1: next tile's score MFMAs interleaved with this tile's softmax;
  // 2: three-stage pipeline (scores of tile j+1, softmax of tile j, P V of tile j-1 in one step)
  static constexpr int PIPE = PIPE_;
  static constexpr bool CAUSAL = CAUSAL_;
  static constexpr int NT = NWAVES * 64;
  static constexpr int BM = NWAVES * 32 * QB;        // query rows per workgroup
  static constexpr int KCH = DQK / 8;                // 16-byte chunks per K-tile row
  static constexpr int VCH = DV / 8;                 // 16-byte chunks per V-tile row
  static constexpr int K_BYTES = BN * DQK * 2;
  static constexpr int V_BYTES = BN * DV * 2;
  static constexpr int STAGE_BYTES = K_BYTES + V_BYTES;
  // Three-stage pipeline: separate rings of K tiles (NKR slots) and V tiles (NVR slots).
  static constexpr int NKR = 3, NVR = 4;
  static constexpr int LDS_BYTES = PIPE == 2 ? NKR * K_BYTES + NVR * V_BYTES : NS * STAGE_BYTES;
  // Direct-load instructions per wave per tile (each moves 64 lanes x 16 bytes).
  static constexpr int K_LOADS = BN * KCH / 64 / NWAVES;
  static constexpr int V_LOADS = BN * VCH / 64 / NWAVES;
  static constexpr int LOADS = K_LOADS + V_LOADS;
  static_assert(DQK % 32 == 0 && DV % 64 == 0, "head dims: d_qk multiple of 32, d_v multiple of 64");
  static_assert(BN % 32 == 0, "key tile must be a multiple of 32");
  static_assert((BN * KCH) % (64 * NWAVES) == 0 && (BN * VCH) % (64 * NWAVES) == 0, "tile split over waves");
  static_assert(NS >= (PIPE ? 3 : 2) && NS <= 5 && LOADS * (NS - 1) < 64, "ring depth");
  static_assert(PIPE != 2 || 2 * V_LOADS + K_LOADS < 64, "vmcnt range");
  static_assert(LDS_BYTES <= 163840, "LDS budget");
};

// One 64-lane direct-to-LDS load of 16 bytes per lane: LDS bytes [lds, lds + 1024) receive the
// lanes' 16 bytes in lane order. Issued as inline asm so that the compiler does not track it: it
// would otherwise assume any later LDS read may alias the in-flight load and wait for every
// outstanding global load first. Completion is ordered explicitly instead (vmcnt wait on the
// issuing wave, then a workgroup barrier) before any wave reads the destination. The SALU write of
// M0 needs one wait state before the load.
__device__ __forceinline__ void dma16_saddr(const void* base, uint32_t voff, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1"
               :
               : "v"(voff), "s"(base), "s"(lds)
               : "memory", "m0");
}
__device__ __forceinline__ void dma16(const void* addr, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off" : : "v"(addr), "s"(lds) : "memory", "m0");
}
__device__ __forceinline__ uint32_t lds_offset(const void* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) void*)p;
}
// Compiler-level memory fence (no instruction): keeps LDS reads on their side of a barrier.
__device__ __forceinline__ void compiler_fence() { asm volatile("" : : : "memory"); }

// Issue this wave's share of the direct-to-LDS loads of one tile: BN rows of CH 16-byte chunks from
// `src` (rows of CH*8 elements, first tile row at key n0) into `stage`. Physical chunk p of the
// stage holds logical chunk (p % CH) ^ swz(row) of row p / CH; rows at or past Sk read row Sk-1
// (their scores are masked, and 0 * finite keeps them out of the accumulator).
template <int NWAVES, int BN, int CH, class Swz>
__device__ __forceinline__ void issue_tile(const uint16_t* __restrict__ src, int n0, int sk, unsigned char* stage,
                                           int wave, int lane, Swz swz) {
  constexpr int NI = BN * CH / 64 / NWAVES;
#pragma unroll
  for (int i = 0; i < NI; ++i) {
    const int blk = wave * NI + i;
    const int pch = blk * 64 + lane;
    const int row = pch / CH;
    const int lch = (pch % CH) ^ swz(row);
    const int key = min(n0 + row, sk - 1);
    dma16(src + (size_t)key * (CH * 8) + lch * 8, lds_offset(stage + blk * 1024));
  }
}

// Per-lane source offsets of this wave's share of a tile, computed once per kernel: a tile that
// lies entirely below Sk is then issued with one address add per load (scalar base = the head's
// first row, kept in SGPRs; 32-bit byte offset per lane = tile offset + lane offset, so one head's
// K or V must span less than 4 GiB, which the API checks); the last, partial tile goes through
// issue_tile, which clamps rows.
template <int NWAVES, int BN, int CH>
struct TileLoader {
  static constexpr int NI = BN * CH / 64 / NWAVES;
  const uint16_t* head;  // wave-uniform
  int off[NI];           // elements from the tile's first row
  template <class Swz>
  __device__ __forceinline__ void init(const uint16_t* head_, int wave, int lane, Swz swz) {
    const uint64_t hb = reinterpret_cast<uint64_t>(head_);
    head = reinterpret_cast<const uint16_t*>(((uint64_t)__builtin_amdgcn_readfirstlane((uint32_t)(hb >> 32)) << 32) |
                                             (uint32_t)__builtin_amdgcn_readfirstlane((uint32_t)hb));
#pragma unroll
    for (int i = 0; i < NI; ++i) {
      const int pch = (wave * NI + i) * 64 + lane;
      const int row = pch / CH;
      off[i] = row * (CH * 8) + ((pch % CH) ^ swz(row)) * 8;
    }
  }
  // Load i of this wave's share of the tile at key n0, which lies entirely below Sk.
  __device__ __forceinline__ void issue_one(int i, int n0, unsigned char* stage, int wave) const {
    dma16_saddr(head, (uint32_t)(n0 * (CH * 8) + off[i]) * 2u, lds_offset(stage + (wave * NI + i) * 1024));
  }
  template <class Swz>
  __device__ __forceinline__ void issue(int n0, int sk, unsigned char* stage, int wave, int lane, Swz swz) const {
    if (n0 + BN <= sk) {
#pragma unroll
      for (int i = 0; i < NI; ++i) issue_one(i, n0, stage, wave);
    } else {
      issue_tile<NWAVES, BN, CH>(head, n0, sk, stage, wave, lane, swz);
    }
  }
};

// Map a hardware workgroup index to (batch, query head, query block). Workgroup t runs on XCD
// t % 8. Logical work items are ordered heaviest query block first (causal), then batch, key/value
// head and group member; each group of `group` consecutive items (the query heads of one key/value
// head at one query block) is placed on one XCD, and groups go to XCDs round-robin.
__device__ __forceinline__ void decode_workgroup(int t, const FwdParams& p, bool causal, int& b, int& hq,
                                                 int& qtile) {
  const int G = p.group;
  const int span = kNumXcd * G;
  const int full = (p.n_wg / span) * span;
  int L = t;
  if (t < full) {
    const int xcd = t % kNumXcd, slot = t / kNumXcd;
    L = ((slot / G) * kNumXcd + xcd) * G + slot % G;
  }
  const int member = L % G;
  int r = L / G;
  const int kvh = r % p.hkv;
  r /= p.hkv;
  b = r % p.batch;
  const int qt = r / p.batch;
  qtile = causal ? p.n_qtiles - 1 - qt : qt;
  hq = kvh * G + member;
}

// Per-wave state and the math of one key/value tile.
template <class C>
struct Attn {
  static constexpr int DQK = C::DQK, DV = C::DV, BN = C::BN, QB = C::QB;
  static constexpr int KS = DQK / 16;  // k-steps of the score product
  static constexpr int KB = BN / 32;   // 32-key blocks per tile
  static constexpr int DB = DV / 32;   // 32-dim blocks of the output
  static constexpr int PS = BN / 16;   // k-steps of the P V product

  typedef f32x16 Scores[KB][QB];

  int i32, h, qw, diag, sk;
  const uint16_t* kg;  // this workgroup's K head in global memory
  float c;
  bool neg;
  int v_key, v_t, v_half;
  bf16x8 qf[QB][KS];
  f32x16 oacc[DB][QB];
  float m_run[QB], l_run[QB];

  // S^T = K Q^T for one tile: per k-step, the K fragments of the 32-key blocks, then KB*QB MFMAs.
  __device__ __forceinline__ void scores(Scores& s, const unsigned char* sK) {
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) {
        const int row = kb * 32 + perm32(i32);
        const u32x4 a = *reinterpret_cast<const u32x4*>(sK + row * (DQK * 2) + (((ks * 2 + h) ^ (i32 & 7)) << 4));
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) {
          if (ks == 0)
            mfma_score_first(s[kb][qb], bit_cast<bf16x8>(a), qf[qb][ks]);
          else
            mfma_score(s[kb][qb], bit_cast<bf16x8>(a), qf[qb][ks]);
        }
      }
    }
#pragma unroll
    for (int kb = 0; kb < KB; ++kb)
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) vgpr_fence(s[kb][qb]);
  }

  // Online softmax of one tile's scores (tile at key n0) and O += V^T P^T from sV.
  __device__ __forceinline__ void softmax_pv(Scores& cur, const unsigned char* sV, int n0, bool masked) {
    if (neg) {
      // scale < 0: scale * s = |scale| * (-s); negation is exact.
#pragma unroll
      for (int kb = 0; kb < KB; ++kb)
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) cur[kb][qb] = -cur[kb][qb];
    }
    float mx[QB];
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      if (masked) {
        const int row = qw + qb * 32 + i32;
        const int last_key = C::CAUSAL ? min(row + diag, sk - 1) : sk - 1;
#pragma unroll
        for (int kb = 0; kb < KB; ++kb)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int key = n0 + kb * 32 + 16 * (r >> 3) + 8 * h + (r & 7);
            if (key > last_key) cur[kb][qb][r] = -INFINITY;
          }
      }
      float m = -INFINITY;
#pragma unroll
      for (int kb = 0; kb < KB; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) m = fmaxf(m, cur[kb][qb][r]);
      mx[qb] = half_swap_max(m) * c;
    }
    // Lazy rescale: the reference maximum m_run moves only when a row's tile maximum exceeds it by
    // more than kRescaleSlack (log2 units), so P <= 2^kRescaleSlack; O and l share the reference,
    // which cancels exactly in O / l. The branch is uniform across the wave.
    bool grow[QB];
    bool any = false;
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      grow[qb] = mx[qb] > m_run[qb] + kRescaleSlack;
      any = any || grow[qb];
    }
    if (__builtin_amdgcn_ballot_w64(any) != 0) {
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) {
        const float m_new = grow[qb] ? mx[qb] : m_run[qb];
        const float alpha = __builtin_amdgcn_exp2f(m_run[qb] - (m_new == -INFINITY ? 0.f : m_new));
        m_run[qb] = m_new;
        l_run[qb] *= alpha;
#pragma unroll
        for (int db = 0; db < DB; ++db) {
          agpr_fence(oacc[db][qb]);
          oacc[db][qb] *= alpha;
          agpr_fence(oacc[db][qb]);
        }
      }
    }
    // exp2, row sums, P -> bf16 (P never leaves the registers it was computed in).
    uint32_t pk[KB][QB][8];
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      const float m_ref = (m_run[qb] == -INFINITY) ? 0.f : m_run[qb];
      float rs = 0.f;
#pragma unroll
      for (int kb = 0; kb < KB; ++kb)
#pragma unroll
        for (int r = 0; r < 16; r += 2) {
          const float e0 = __builtin_amdgcn_exp2f(fmaf(cur[kb][qb][r], c, -m_ref));
          const float e1 = __builtin_amdgcn_exp2f(fmaf(cur[kb][qb][r + 1], c, -m_ref));
          rs += e0 + e1;
          pk[kb][qb][r >> 1] = pack_bf16x2(e0, e1);
        }
      l_run[qb] += rs;
    }
    // O^T += V^T P^T
#pragma unroll
    for (int ps = 0; ps < PS; ++ps) {
      bf16x8 pb[QB];
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) {
        const int kb = ps >> 1, base = (ps & 1) * 4;
        const u32x4 w = {pk[kb][qb][base], pk[kb][qb][base + 1], pk[kb][qb][base + 2], pk[kb][qb][base + 3]};
        pb[qb] = bit_cast<bf16x8>(w);
      }
#pragma unroll
      for (int db = 0; db < DB; ++db) {
        // A operand V^T[dims db*32 + 0..31][keys 16*ps + 0..15]: lane (group G, slot j) points the
        // transpose read at key 16*ps + 8*(G/2) + j/4 (then +4), dims db*32 + 16*(G%2) + 4*(j%4).
        const unsigned char* base = sV + (ps * 16 + v_key) * (DV * 2) + (((db * 4) ^ v_t) << 4) + v_half;
        const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(base));
        const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(base + 4 * DV * 2));
        const i16x8 a = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) mfma_out(oacc[db][qb], bit_cast<bf16x8>(a), pb[qb]);
      }
    }
  }

  // ---- software-pipelined step ---------------------------------------------------------------
  // Tile j's softmax and P V, with tile j+1's score MFMAs interleaved into the softmax. The order
  // of MFMAs, VALU chunks and LDS reads is fixed with scheduling fences so that one wave per SIMD
  // keeps the MFMA unit busy while it does the softmax arithmetic.
  static constexpr int NMS = KS * KB * QB;                        // score MFMAs per tile
  static constexpr int N1 = (NMS / 4 > KB * QB) ? NMS / 4 : KB * QB;  // of them before the rescale branch
  static constexpr int NE = QB * KB * 16;                          // score elements per lane
  static constexpr int KPF = 2;                                    // k-steps of K fragments read ahead
  static constexpr int VPF = 2;                                    // V fragments read ahead

  __device__ __forceinline__ u32x4 kfrag(const unsigned char* sK, int ks, int kb) const {
    const int row = kb * 32 + perm32(i32);
    return *reinterpret_cast<const u32x4*>(sK + row * (DQK * 2) + (((ks * 2 + h) ^ (i32 & 7)) << 4));
  }
  __device__ __forceinline__ bf16x8 vfrag(const unsigned char* sV, int ps, int db) const {
    const unsigned char* base = sV + (ps * 16 + v_key) * (DV * 2) + (((db * 4) ^ v_t) << 4) + v_half;
    const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(base));
    const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(base + 4 * DV * 2));
    return bit_cast<bf16x8>(__builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
  }

  __device__ __forceinline__ void step_pipelined(Scores& cur, Scores& nxt, const unsigned char* sKn,
                                                 const unsigned char* sVc, int n0, bool masked) {
    if (neg) {
#pragma unroll
      for (int kb = 0; kb < KB; ++kb)
#pragma unroll
        for (int qb = 0; qb < QB; ++qb) cur[kb][qb] = -cur[kb][qb];
    }
    if (masked) {
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) {
        const int row = qw + qb * 32 + i32;
        const int last_key = C::CAUSAL ? min(row + diag, sk - 1) : sk - 1;
#pragma unroll
        for (int kb = 0; kb < KB; ++kb)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int key = n0 + kb * 32 + 16 * (r >> 3) + 8 * h + (r & 7);
            if (key > last_key) cur[kb][qb][r] = -INFINITY;
          }
      }
    }
    u32x4 kf[KS][KB];
#pragma unroll
    for (int ks = 0; ks < KPF && ks < KS; ++ks)
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) kf[ks][kb] = kfrag(sKn, ks, kb);
    __builtin_amdgcn_sched_barrier(0);

    // -- phase A1: score MFMAs 0..N1-1 with the row maxima
    float m[QB];
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) m[qb] = -INFINITY;
#pragma unroll
    for (int i = 0; i < N1; ++i) {
      score_mfma(nxt, kf, sKn, i);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int e = 0; e < NE; ++e)
        if (e * N1 / NE == i) {
          const int qb = e / (KB * 16), kb = (e / 16) % KB, r = e % 16;
          m[qb] = fmaxf(m[qb], cur[kb][qb][r]);
        }
      __builtin_amdgcn_sched_barrier(0);
    }
#if FA_SCORE_BUILTIN
#pragma unroll
    for (int i = 0; i < N1; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x002, 4, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    }
#endif
    float mx[QB];
    bool grow[QB];
    bool any = false;
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      mx[qb] = half_swap_max(m[qb]) * c;
      grow[qb] = mx[qb] > m_run[qb] + kRescaleSlack;
      any = any || grow[qb];
    }
    // Lazy rescale (see softmax_pv); rare and uniform across the wave.
    if (__builtin_amdgcn_ballot_w64(any) != 0) {
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) {
        const float m_new = grow[qb] ? mx[qb] : m_run[qb];
        const float alpha = __builtin_amdgcn_exp2f(m_run[qb] - (m_new == -INFINITY ? 0.f : m_new));
        m_run[qb] = m_new;
        l_run[qb] *= alpha;
#pragma unroll
        for (int db = 0; db < DB; ++db) {
          agpr_fence(oacc[db][qb]);
          oacc[db][qb] *= alpha;
          agpr_fence(oacc[db][qb]);
        }
      }
    }
    float m_ref[QB], rs[QB];
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      m_ref[qb] = (m_run[qb] == -INFINITY) ? 0.f : m_run[qb];
      rs[qb] = 0.f;
    }
    __builtin_amdgcn_sched_barrier(0);

    // -- phase A2: score MFMAs N1..NMS-1 with exp2, row sums and P -> bf16
    uint32_t pk[KB][QB][8];
    constexpr int NC = NMS - N1, NP = NE / 2;
#pragma unroll
    for (int i = N1; i < NMS; ++i) {
      score_mfma(nxt, kf, sKn, i);
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int pp = 0; pp < NP; ++pp)
        if (pp * NC / NP == i - N1) {
          const int e = 2 * pp;
          const int qb = e / (KB * 16), kb = (e / 16) % KB, r = e % 16;
          const float e0 = __builtin_amdgcn_exp2f(fmaf(cur[kb][qb][r], c, -m_ref[qb]));
          const float e1 = __builtin_amdgcn_exp2f(fmaf(cur[kb][qb][r + 1], c, -m_ref[qb]));
          rs[qb] += e0 + e1;
          pk[kb][qb][r >> 1] = pack_bf16x2(e0, e1);
        }
      __builtin_amdgcn_sched_barrier(0);
    }
#if FA_SCORE_BUILTIN
#pragma unroll
    for (int i = N1; i < NMS; ++i) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x002, 8, 0);
      __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
    }
#endif
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) l_run[qb] += rs[qb];

    // -- phase B: O^T += V^T P^T, V fragments read VPF steps ahead; the next tile's scores move into
    //    `cur` once their MFMAs are long finished (after the first 4 P V MFMAs).
    constexpr int NV = PS * DB;
    bf16x8 vf[NV];
#pragma unroll
    for (int t = 0; t < VPF && t < NV; ++t) vf[t] = vfrag(sVc, t / DB, t % DB);
    __builtin_amdgcn_sched_barrier(0);
    constexpr int NCOPY = KB * QB;
#pragma unroll
    for (int t = 0; t < NV; ++t) {
      const int ps = t / DB, db = t % DB;
      if (t + VPF < NV) vf[t + VPF] = vfrag(sVc, (t + VPF) / DB, (t + VPF) % DB);
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) {
        const int kb = ps >> 1, base = (ps & 1) * 4;
        const u32x4 w = {pk[kb][qb][base], pk[kb][qb][base + 1], pk[kb][qb][base + 2], pk[kb][qb][base + 3]};
        mfma_out(oacc[db][qb], vf[t], bit_cast<bf16x8>(w));
      }
      __builtin_amdgcn_sched_barrier(0);
      if (t >= 4 && t - 4 < NCOPY) {
        const int cc = t - 4;
        cur[cc / QB][cc % QB] = nxt[cc / QB][cc % QB];
      }
      __builtin_amdgcn_sched_barrier(0);
    }
#pragma unroll
    for (int cc = (NV - 4 > 0 ? NV - 4 : 0); cc < NCOPY; ++cc) cur[cc / QB][cc % QB] = nxt[cc / QB][cc % QB];
  }

  // Score MFMA number i of a tile (order ks, kb, qb), reading K fragments KPF k-steps ahead.
  __device__ __forceinline__ void score_mfma(Scores& s, u32x4 (&kf)[KS][KB], const unsigned char* sK, int i) {
    const int ks = i / (KB * QB), kb = (i / QB) % KB, qb = i % QB;
    if (kb == 0 && qb == 0 && ks + KPF < KS) {
#pragma unroll
      for (int kb2 = 0; kb2 < KB; ++kb2) kf[ks + KPF][kb2] = kfrag(sK, ks + KPF, kb2);
    }
#if FA_SCORE_BUILTIN
    s[kb][qb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bit_cast<bf16x8>(kf[ks][kb]), qf[qb][ks],
                                                        ks == 0 ? f32x16{} : s[kb][qb], 0, 0, 0);
#else
    if (ks == 0)
      mfma_score_first(s[kb][qb], bit_cast<bf16x8>(kf[ks][kb]), qf[qb][ks]);
    else
      mfma_score(s[kb][qb], bit_cast<bf16x8>(kf[ks][kb]), qf[qb][ks]);
#endif
  }

  // ---- three-stage pipeline -------------------------------------------------------------------
  // One step works on three key tiles at once: the score MFMAs of tile j+1 (K from LDS), the
  // exponentials of tile j (VALU, scores computed in the previous step) and the P V MFMAs of tile
  // j-1 (V from LDS, P packed in the previous step). Nothing inside a step depends on anything
  // else inside it, so the two kinds of MFMA alternate and the softmax arithmetic is spread evenly
  // over all of them: a single wave per SIMD then keeps the matrix unit fed while it issues VALU.
  //
  // Reference maximum: tile 0 sets m_run to the exact row maximum. Afterwards the per-element
  // maximum is not computed at all: each lane's sum of its tile exponentials bounds every one of
  // them, so when all lane sums stay <= 2^kRescaleSlack no probability exceeds 2^kRescaleSlack and
  // the step is final. Otherwise (rare: a new maximum well above the reference) the step is redone
  // for that tile from its exact row maximum (rebase), with O and l rescaled, as in Alg. 1.
  typedef uint32_t Probs[KB][QB][8];                 // P of one tile as packed bf16 pairs
  static constexpr int NMP = PS * DB * QB;            // P V MFMAs per tile
  static constexpr int NSL = NMS + NMP;               // MFMA slots per step
  static constexpr int NEP = KB * QB * 8;             // exponential pairs per lane per tile
  static constexpr int NVF = PS * DB;                 // V fragments per tile

  float cs;        // scale * log2(e), signed
  float mask_val;  // a score that cs maps to -inf

  // Slot order: the P V MFMAs of tile j-1 first, then the score MFMAs of tile j+1. The
  // exponentials of tile j run from slot E0 on, evenly spread: P V consumes the previous tile's P
  // chunk c (16 keys) in slots [c*E0, (c+1)*E0), and chunk c of the new P is produced only after
  // that, so both tiles' P share registers. The score accumulators of block kb+1 start after
  // the exponentials of block kb of the previous scores (block-major order), so the two score
  // tiles overlap in registers only partly.
#if FA_ORDER
  static constexpr int E0 = NMP / PS;
  static_assert(NSL >= 5 * E0, "exponentials of chunk c must follow the P V MFMAs of chunk c");
  static constexpr bool slot_is_score(int sl) { return sl >= NMP; }
  static constexpr int slot_score(int sl) { return sl - NMP; }
  static constexpr int slot_pv(int sl) { return sl; }
#else
  static constexpr int E0 = 0;
  static constexpr bool slot_is_score(int sl) { return (sl + 1) * NMS / NSL > sl * NMS / NSL; }
  static constexpr int slot_score(int sl) { return sl * NMS / NSL; }
  static constexpr int slot_pv(int sl) { return sl - sl * NMS / NSL; }
#endif
  // exponential pairs of slot sl: u with E0 + floor(u * (NSL - E0) / NEP) == sl
  static constexpr int exp_begin(int sl) { return sl < E0 ? 0 : ((sl - E0) * NEP + NSL - E0 - 1) / (NSL - E0); }
  static constexpr int exp_end(int sl) { return sl < E0 ? 0 : ((sl - E0 + 1) * NEP + NSL - E0 - 1) / (NSL - E0); }

  // Score MFMA number i of a tile in 32-key-block-major order (kb, ks, qb): the accumulators of
  // block kb+1 start only when block kb is finished, and the exponentials consume the previous
  // tile's scores in the same block order, so the two score tiles share registers. K fragments
  // (sequence f = kb*KS + ks) are read KPF ahead.
  __device__ __forceinline__ void score_mfma_kb(Scores& s, u32x4 (&kf)[KB * KS], const unsigned char* sK, int i) {
    const int kb = i / (KS * QB), ks = (i / QB) % KS, qb = i % QB, f = kb * KS + ks;
    if (qb == 0 && f + KPF < KB * KS) kf[f + KPF] = kfrag(sK, (f + KPF) % KS, (f + KPF) / KS);
    s[kb][qb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bit_cast<bf16x8>(kf[f]), qf[qb][ks],
                                                        ks == 0 ? f32x16{} : s[kb][qb], 0, 0, 0);
  }

  // Masked keys of tile n0 (key > i + diag, or key >= Sk) get mask_val.
  __device__ __forceinline__ void mask_tile(Scores& s, int n0) const {
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      const int row = qw + qb * 32 + i32;
      const int last_key = C::CAUSAL ? min(row + diag, sk - 1) : sk - 1;
      const int lim = last_key - n0 - 8 * h;  // key offset kb*32 + 16*(r/8) + r%8 is masked iff > lim
#pragma unroll
      for (int kb = 0; kb < KB; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          if (kb * 32 + 16 * (r >> 3) + (r & 7) > lim) s[kb][qb][r] = mask_val;
    }
  }

  // Exact maximum of cs * score over the row (both lane halves), -inf if every key is masked.
  __device__ __forceinline__ float row_max(const Scores& s, int qb) const {
    float m = -INFINITY;
#pragma unroll
    for (int kb = 0; kb < KB; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) m = fmaxf(m, s[kb][qb][r] * cs);
    return half_swap_max(m);
  }

  // Exponential pair u of a tile: p = 2^(cs * s - m_ref), the lane's row sum, and the bf16 pair.
  __device__ __forceinline__ void exp_pair(int u, const Scores& cur, Probs& pk, const float (&mref)[QB],
                                           float (&rs)[QB]) const {
    const int qb = u % QB, rp = (u / QB) % 8, kb = u / (QB * 8);
    const float e0 = __builtin_amdgcn_exp2f(fmaf(cur[kb][qb][2 * rp], cs, -mref[qb]));
    const float e1 = __builtin_amdgcn_exp2f(fmaf(cur[kb][qb][2 * rp + 1], cs, -mref[qb]));
    rs[qb] += e0 + e1;
    pk[kb][qb][rp] = pack_bf16x2(e0, e1);
    // Keep the pack here: otherwise it is sunk past the rebase branch, which keeps both fp32
    // exponentials alive across the whole step.
    asm volatile("" : "+v"(pk[kb][qb][rp]));
  }

  // P V MFMA number p of a tile (order ps, db, qb), V fragments read VPF ahead.
  __device__ __forceinline__ void pv_mfma(int p, const Probs& pk, bf16x8 (&vf)[NVF], const unsigned char* sV) {
    const int t = p / QB, qb = p % QB, ps = t / DB, db = t % DB;
    if (qb == 0 && t + VPF < NVF) vf[t + VPF] = vfrag(sV, (t + VPF) / DB, (t + VPF) % DB);
    const int kb = ps >> 1, base = (ps & 1) * 4;
    const u32x4 w = {pk[kb][qb][base], pk[kb][qb][base + 1], pk[kb][qb][base + 2], pk[kb][qb][base + 3]};
    mfma_out(oacc[db][qb], vf[t], bit_cast<bf16x8>(w));
  }

  // All P V MFMAs of one tile (the last tile, after the loop).
  __device__ __forceinline__ void pv_tile(const Probs& pk, const unsigned char* sV) {
    bf16x8 vf[NVF];
#pragma unroll
    for (int t = 0; t < VPF && t < NVF; ++t) vf[t] = vfrag(sV, t / DB, t % DB);
#pragma unroll
    for (int pi = 0; pi < NMP; ++pi) pv_mfma(pi, pk, vf, sV);
  }

  // Redo a tile's exponentials from its exact row maximum; O and l follow the new reference. The
  // tile's scores are recomputed from K in global memory (kg, rows clamped to Sk-1): by the end of
  // the step the raw scores are gone and the tile's LDS slot holds a later tile. Rare by design.
  __device__ __forceinline__ void rebase(Probs& pk, float (&rs)[QB], int n0, bool masked) {
    Scores cur;
#pragma unroll
    for (int kb = 0; kb < KB; ++kb) {
      const int row = min(n0 + kb * 32 + perm32(i32), sk - 1);
      const uint16_t* krow = kg + (size_t)row * DQK + 8 * h;
#pragma unroll
      for (int ks = 0; ks < KS; ++ks) {
        const u32x4 a = *reinterpret_cast<const u32x4*>(krow + 16 * ks);
#pragma unroll
        for (int qb = 0; qb < QB; ++qb)
          cur[kb][qb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bit_cast<bf16x8>(a), qf[qb][ks],
                                                                ks == 0 ? f32x16{} : cur[kb][qb], 0, 0, 0);
      }
    }
    if (masked) mask_tile(cur, n0);
    float mref[QB];
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      const float m_new = fmaxf(m_run[qb], row_max(cur, qb));
      const float alpha = m_new == -INFINITY ? 1.f : __builtin_amdgcn_exp2f(m_run[qb] - m_new);
      m_run[qb] = m_new;
      l_run[qb] *= alpha;
#pragma unroll
      for (int db = 0; db < DB; ++db) {
        agpr_fence(oacc[db][qb]);
        oacc[db][qb] *= alpha;
        agpr_fence(oacc[db][qb]);
      }
      mref[qb] = m_new == -INFINITY ? 0.f : m_new;
      rs[qb] = 0.f;
    }
#pragma unroll
    for (int u = 0; u < NEP; ++u) exp_pair(u, cur, pk, mref, rs);
  }

  // `issue(k)` starts direct-to-LDS load k (0 <= k < LOADS) of the tiles this step prefetches; the
  // loads are spread over the step, one every NSL / LOADS MFMA slots.
  template <class Issue>
  __device__ __forceinline__ void step3(Scores& cur, Scores& nxt, Probs& pk_new, const Probs& pk_old,
                                        const unsigned char* sKn, const unsigned char* sVo, bool masked, int n0,
                                        Issue&& issue) {
    if (masked) mask_tile(cur, n0);
    float mref[QB], rs[QB];
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      mref[qb] = m_run[qb] == -INFINITY ? 0.f : m_run[qb];
      rs[qb] = 0.f;
    }
    u32x4 kf[KB * KS];
#pragma unroll
    for (int f = 0; f < KPF && f < KB * KS; ++f) kf[f] = kfrag(sKn, f % KS, f / KS);
    bf16x8 vf[NVF];
#pragma unroll
    for (int t = 0; t < VPF && t < NVF; ++t) vf[t] = vfrag(sVo, t / DB, t % DB);
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int sl = 0; sl < NSL; ++sl) {
      constexpr int SPREAD = NSL / C::LOADS;
      if (sl % SPREAD == 0 && sl / SPREAD < C::LOADS) issue(sl / SPREAD);
      if (slot_is_score(sl))
        score_mfma_kb(nxt, kf, sKn, slot_score(sl));
      else
        pv_mfma(slot_pv(sl), pk_old, vf, sVo);
#pragma unroll
      for (int u = exp_begin(sl); u < exp_end(sl); ++u) exp_pair(u, cur, pk_new, mref, rs);
      __builtin_amdgcn_sched_barrier(0);
    }
    bool over = false;
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) over = over || !(rs[qb] <= kOverflowSum);
    if (__builtin_amdgcn_ballot_w64(over) != 0) rebase(pk_new, rs, n0, masked);
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) l_run[qb] += rs[qb];
  }
};

template <class C>
__global__ __attribute__((amdgpu_flat_work_group_size(C::NT, C::NT), amdgpu_waves_per_eu(C::WPE, C::WPE)))
void fa_fwd_kernel(FwdParams p) {
  using A = Attn<C>;
  constexpr int DQK = C::DQK, DV = C::DV, BN = C::BN, QB = C::QB, NS = C::NS;

  __shared__ __attribute__((aligned(1024))) unsigned char smem[C::LDS_BYTES];
  auto stage_k = [&](int s) { return smem + s * C::STAGE_BYTES; };  // rings of the one- and two-stage loops
  auto stage_v = [&](int s) { return smem + s * C::STAGE_BYTES + C::K_BYTES; };
  auto kswz = [](int row) { return k_swizzle(row); };
  auto vswz = [](int row) { return v_swizzle(row); };

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  A st;
  st.i32 = lane & 31;
  st.h = lane >> 5;
  // Lane constants of the V transpose read: group G = lane/16, slot j = lane%16.
  st.v_key = 8 * (lane >> 5) + ((lane & 15) >> 2);                             // key in the 16-key step
  st.v_t = (2 * ((lane >> 4) & 1) + ((lane & 3) >> 1)) ^ v_swizzle(st.v_key);  // low chunk bits, swizzled
  st.v_half = (lane & 1) * 8;                                                  // byte offset in the chunk
  st.c = p.c;
  st.neg = p.qsign != 0;
  st.sk = p.sk;

  int b, hq, qtile;
  decode_workgroup(blockIdx.x, p, C::CAUSAL, b, hq, qtile);
  const int g = hq / p.group;
  const uint16_t* __restrict__ qh = p.q + (size_t)(b * p.hq + hq) * p.sq * DQK;
  const uint16_t* __restrict__ kh = p.k + (size_t)(b * p.hkv + g) * p.sk * DQK;
  const uint16_t* __restrict__ vh = p.v + (size_t)(b * p.hkv + g) * p.sk * DV;
  st.kg = kh;

  const int q0 = qtile * C::BM;
  st.qw = q0 + wave * 32 * QB;  // first query row of this wave
  st.diag = p.sk - p.sq;        // key j is visible to query i iff j <= i + diag

  // Key tiles this workgroup visits, and how many leading ones need no mask for any of its rows.
  int kv_end = p.sk;
  int n_plain = p.sk / BN;
  if (C::CAUSAL) {
    const int last_row = min(q0 + C::BM, p.sq) - 1;
    kv_end = max(0, min(p.sk, last_row + st.diag + 1));
    n_plain = min(n_plain, max(0, q0 + st.diag + 1) / BN);
  }
  const int nt = (kv_end + BN - 1) / BN;

  // Three-stage pipeline: K tiles in a ring of NKR slots, V tiles in a ring of NVR slots. Step j
  // issues K(j+3) and V(j+2); the prologue issues the same groups for j = -3, -2, -1, i.e.
  // K0, K1, V0, K2, V1 in this order.
  TileLoader<C::NWAVES, BN, C::KCH> kload;
  TileLoader<C::NWAVES, BN, C::VCH> vload;
  auto kslot = [&](int t) { return smem + (t % C::NKR) * C::K_BYTES; };
  auto vslot = [&](int t) { return smem + C::NKR * C::K_BYTES + (t % C::NVR) * C::V_BYTES; };
  auto issue_group = [&](int j) {
    if (j + 3 < nt) kload.issue((j + 3) * BN, p.sk, kslot(j + 3), wave, lane, kswz);
    if (j + 2 >= 0 && j + 2 < nt) vload.issue((j + 2) * BN, p.sk, vslot(j + 2), wave, lane, vswz);
  };
  if (C::PIPE == 2) {
    kload.init(kh, wave, lane, kswz);
    vload.init(vh, wave, lane, vswz);
    issue_group(-3);
    issue_group(-2);
    issue_group(-1);
  } else {
    // Start the first NS-1 tiles, then load Q while they are in flight.
    for (int t = 0; t < NS - 1 && t < nt; ++t) {
      issue_tile<C::NWAVES, BN, C::KCH>(kh, t * BN, p.sk, stage_k(t), wave, lane, kswz);
      issue_tile<C::NWAVES, BN, C::VCH>(vh, t * BN, p.sk, stage_v(t), wave, lane, vswz);
    }
  }

  // Q rows of this wave as B operands of the score product, resident in AGPRs: lane (i32, h) holds
  // row qw+32*qb+i32, dims 16*ks + 8*h .. +7. Rows past Sq read row Sq-1 instead; their outputs are
  // never stored. (load_q waits for all of this wave's loads, tiles included.)
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    const int row = min(st.qw + qb * 32 + st.i32, p.sq - 1);
#pragma unroll
    for (int ks = 0; ks < A::KS; ++ks) st.qf[qb][ks] = load_q(qh + (size_t)row * DQK + ks * 16 + st.h * 8);
  }

#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    st.m_run[qb] = -INFINITY;
    st.l_run[qb] = 0.f;
#pragma unroll
    for (int db = 0; db < A::DB; ++db) {
      st.oacc[db][qb] = f32x16{};
      agpr_fence(st.oacc[db][qb]);
    }
  }

  if (C::PIPE == 2) {
    st.cs = st.neg ? -st.c : st.c;
    st.mask_val = st.neg ? INFINITY : -INFINITY;
    typename A::Scores sA, sB;
    typename A::Probs pA, pB;
    if (nt > 0) {
      // Tile 0: scores, mask, exact row maxima. P of "tile -1" is zero (its P V step reads the
      // finite V tile 0 and adds nothing).
      compiler_fence();
      __builtin_amdgcn_s_barrier();
      compiler_fence();
      st.scores(sA, kslot(0));
      if (n_plain == 0) st.mask_tile(sA, 0);
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) st.m_run[qb] = st.row_max(sA, qb);
#pragma unroll
      for (int kb = 0; kb < A::KB; ++kb)
#pragma unroll
        for (int qb = 0; qb < QB; ++qb)
#pragma unroll
          for (int r = 0; r < 8; ++r) pB[kb][qb][r] = 0u;
    }
    // Before step j: K(j+1) and V(j-1) must have landed. This wave's loads issued after K(j+1) are
    // V(j), K(j+2) (if it exists) and V(j+1); on the last step only V(j) follows V(j-1).
    // Loads of group j: a tile that lies entirely below Sk is deferred and issued load by load
    // inside step j; a partial last tile is issued at once here (the order K, V of the group is
    // kept: when V(j+2) is partial, K(j+3) does not exist).
    int gj = 0;                        // group being issued (uniform)
    bool kdefer = false, vdefer = false;
    auto issue_k = [&](int k) {
      if (k < C::K_LOADS) {
        if (kdefer) kload.issue_one(k, (gj + 3) * BN, kslot(gj + 3), wave);
      } else {
        if (vdefer) vload.issue_one(k - C::K_LOADS, (gj + 2) * BN, vslot(gj + 2), wave);
      }
    };
    auto start_group = [&](int j) {
      gj = j;
      kdefer = vdefer = false;
      if (j + 3 < nt) {
        if ((j + 4) * BN <= p.sk && FA_SPREAD)
          kdefer = true;
        else
          kload.issue((j + 3) * BN, p.sk, kslot(j + 3), wave, lane, kswz);
      }
      if (j + 2 < nt) {
        if ((j + 3) * BN <= p.sk && FA_SPREAD)
          vdefer = true;
        else
          vload.issue((j + 2) * BN, p.sk, vslot(j + 2), wave, lane, vswz);
      }
    };
    auto sync_step = [&](int j) {
      if (j + 1 < nt) {
        if (j + 2 < nt)
          wait_vmcnt<2 * C::V_LOADS + C::K_LOADS>();
        else
          wait_vmcnt<2 * C::V_LOADS>();
      } else {
        wait_vmcnt<C::V_LOADS>();
      }
      compiler_fence();
      __builtin_amdgcn_s_barrier();
      compiler_fence();
      start_group(j);
    };
    int j = 0;
    for (; j + 1 < nt; j += 2) {
      sync_step(j);
      st.step3(sA, sB, pA, pB, kslot(j + 1), vslot(j > 0 ? j - 1 : 0), j > 0 && j >= n_plain, j * BN, issue_k);
      sync_step(j + 1);
      st.step3(sB, sA, pB, pA, kslot(j + 2), vslot(j), j + 1 >= n_plain, (j + 1) * BN, issue_k);
    }
    if (j < nt) {
      sync_step(j);
      st.step3(sA, sB, pA, pB, kslot(j + 1), vslot(j > 0 ? j - 1 : 0), j > 0 && j >= n_plain, j * BN, issue_k);
    }
    if (nt > 0) {
      // P V of the last tile.
      wait_vmcnt<0>();
      compiler_fence();
      __builtin_amdgcn_s_barrier();
      compiler_fence();
      // One call on a selected copy of P: two calls would leave O in different registers and the
      // copies that merge them could read MFMA results before they are written.
      // (The select is a bit mask: a ternary on the elements would be folded into a select of the
      // two arrays' addresses, which forces both into scratch memory.)
      typename A::Probs pl;
      const uint32_t take_a = (nt & 1) ? 0xffffffffu : 0u;
#pragma unroll
      for (int kb = 0; kb < A::KB; ++kb)
#pragma unroll
        for (int qb = 0; qb < QB; ++qb)
#pragma unroll
          for (int r = 0; r < 8; ++r) pl[kb][qb][r] = (pA[kb][qb][r] & take_a) | (pB[kb][qb][r] & ~take_a);
      st.pv_tile(pl, vslot(nt - 1));
#pragma unroll
      for (int qb = 0; qb < QB; ++qb)
#pragma unroll
        for (int db = 0; db < A::DB; ++db) agpr_fence(st.oacc[db][qb]);
    }
  } else if (C::PIPE) {
    // Pipelined loop: iteration j reads K_{j+1} and V_j. The prologue has already waited for all of
    // this wave's loads (load_q); the barrier publishes tiles 0..NS-2 and the scores of tile 0 are
    // computed up front.
    typename A::Scores cur, nxt;
    if (nt > 0) {
      __builtin_amdgcn_s_barrier();
      st.scores(cur, stage_k(0));
    }
    for (int j = 0; j < nt; ++j) {
      // Tile j+1 must be complete: at most (tiles issued after it) * LOADS loads may be outstanding.
      const int issued = min(nt - 1, j + NS - 2);
      const int later = issued - min(j + 1, nt - 1);
      if (NS >= 5 && later >= 2)
        wait_vmcnt<(NS >= 5 ? 2 : 0) * C::LOADS>();
      else if (NS >= 4 && later >= 1)
        wait_vmcnt<(NS >= 4 ? 1 : 0) * C::LOADS>();
      else
        wait_vmcnt<0>();
      __builtin_amdgcn_s_barrier();
      if (j + NS - 1 < nt) {
        const int s = (j + NS - 1) % NS;
        issue_tile<C::NWAVES, BN, C::KCH>(kh, (j + NS - 1) * BN, p.sk, stage_k(s), wave, lane, kswz);
        issue_tile<C::NWAVES, BN, C::VCH>(vh, (j + NS - 1) * BN, p.sk, stage_v(s), wave, lane, vswz);
      }
      st.step_pipelined(cur, nxt, stage_k((j + 1) % NS), stage_v(j % NS), j * BN, j >= n_plain);
    }
  } else
  for (int j = 0; j < nt; ++j) {
    // This wave's loads of tile j are complete once at most (tiles issued after it) * LOADS of its
    // loads are outstanding; the barrier then publishes every wave's part of tile j and guarantees
    // that every wave is done with tile j-1, whose stage the next issue overwrites.
    const int later = min(nt - 1, j + NS - 2) - j;
    if (NS >= 4 && later >= 2)
      wait_vmcnt<(NS >= 4 ? 2 : 0) * C::LOADS>();
    else if (NS >= 3 && later >= 1)
      wait_vmcnt<(NS >= 3 ? 1 : 0) * C::LOADS>();
    else
      wait_vmcnt<0>();
    __builtin_amdgcn_s_barrier();
    if (j + NS - 1 < nt) {
      const int s = (j + NS - 1) % NS;
      issue_tile<C::NWAVES, BN, C::KCH>(kh, (j + NS - 1) * BN, p.sk, stage_k(s), wave, lane, kswz);
      issue_tile<C::NWAVES, BN, C::VCH>(vh, (j + NS - 1) * BN, p.sk, stage_v(s), wave, lane, vswz);
    }
    const int s = j % NS;
    typename A::Scores sc;
    st.scores(sc, stage_k(s));
    st.softmax_pv(sc, stage_v(s), j * BN, j >= n_plain);
  }

  // ---- epilogue: O = acc / l, LSE = ln 2 * (m + log2 l) ---------------------------------------
#pragma unroll
  for (int qb = 0; qb < QB; ++qb)
#pragma unroll
    for (int db = 0; db < A::DB; ++db) agpr_fence(st.oacc[db][qb]);
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    const float l_tot = half_swap_sum(st.l_run[qb]);
    const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
    const int row = st.qw + qb * 32 + st.i32;
    if (row < p.sq) {
      uint16_t* orow = p.o + ((size_t)(b * p.hq + hq) * p.sq + row) * DV;
#pragma unroll
      for (int db = 0; db < A::DB; ++db)
#pragma unroll
        for (int g4 = 0; g4 < 4; ++g4) {
          const int d = db * 32 + 8 * g4 + 4 * st.h;
          const u32x2 w = {pack_bf16x2(st.oacc[db][qb][4 * g4] * inv, st.oacc[db][qb][4 * g4 + 1] * inv),
                           pack_bf16x2(st.oacc[db][qb][4 * g4 + 2] * inv, st.oacc[db][qb][4 * g4 + 3] * inv)};
          *reinterpret_cast<u32x2*>(orow + d) = w;
        }
      if (p.lse != nullptr && st.h == 0)
        p.lse[(size_t)(b * p.hq + hq) * p.sq + row] =
            l_tot > 0.f ? (st.m_run[qb] + log2f(l_tot)) * kLn2 : -INFINITY;
    }
  }
}

// Tile configuration (compile-time): key-tile width, waves per workgroup, 32-row query blocks per
// wave, target waves per SIMD, and LDS ring depth.
#ifndef FA_BN
#define FA_BN 64
#endif
#ifndef FA_NWAVES
#define FA_NWAVES 4
#endif
#ifndef FA_QB
#define FA_QB 2
#endif
#ifndef FA_WPE
#define FA_WPE 1
#endif
#ifndef FA_NS
#define FA_NS 4
#endif
#ifndef FA_PIPE
#define FA_PIPE 2
#endif


template <int DQK, int DV, bool CAUSAL>
struct Instance {
  // Ring depth: FA_NS stages, fewer if that many do not fit in LDS.
  static constexpr int STAGE = FA_BN * (DQK + DV) * 2;
  static constexpr int NS = (FA_NS * STAGE <= 163840) ? FA_NS : 163840 / STAGE;
  using C = Cfg<DQK, DV, FA_BN, FA_NWAVES, FA_QB, FA_WPE, NS, FA_PIPE, CAUSAL>;
};

template <int DQK, int DV, bool CAUSAL>
hipError_t launch_instance(FwdParams p, hipStream_t stream) {
  using C = typename Instance<DQK, DV, CAUSAL>::C;
  p.n_qtiles = (p.sq + C::BM - 1) / C::BM;
  p.n_wg = p.batch * p.hq * p.n_qtiles;
  void* args[] = {&p};
  return hipLaunchKernel(reinterpret_cast<const void*>(&fa_fwd_kernel<C>), dim3(p.n_wg), dim3(C::NT), args, 0,
                         stream);
}

}  // namespace

int block_rows(int d_qk, int d_v, bool causal) {
  (void)causal;
  if (d_qk == 64 && d_v == 64) return Instance<64, 64, false>::C::BM;
  if (d_qk == 128 && d_v == 128) return Instance<128, 128, false>::C::BM;
  if (d_qk == 192 && d_v == 128) return Instance<192, 128, false>::C::BM;
  return 0;
}

hipError_t launch_forward(FwdParams p, int d_qk, int d_v, bool causal, hipStream_t stream) {
  if (d_qk == 64 && d_v == 64) return causal ? launch_instance<64, 64, true>(p, stream) : launch_instance<64, 64, false>(p, stream);
  if (d_qk == 128 && d_v == 128)
    return causal ? launch_instance<128, 128, true>(p, stream) : launch_instance<128, 128, false>(p, stream);
  if (d_qk == 192 && d_v == 128)
    return causal ? launch_instance<192, 128, true>(p, stream) : launch_instance<192, 128, false>(p, stream);
  return hipErrorInvalidValue;
}

}  // namespace fa
