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

constexpr float kLn2 = 0.69314718055994530942f;
constexpr float kRescaleSlack = 8.0f;
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

template <int DQK_, int DV_, int BN_, int NWAVES_, int QB_, int WPE_, int NS_, bool CAUSAL_>
struct Cfg {
  static constexpr int DQK = DQK_, DV = DV_, BN = BN_, NWAVES = NWAVES_, QB = QB_, WPE = WPE_, NS = NS_;
  static constexpr bool CAUSAL = CAUSAL_;
  static constexpr int NT = NWAVES * 64;
  static constexpr int BM = NWAVES * 32 * QB;        // query rows per workgroup
  static constexpr int KCH = DQK / 8;                // 16-byte chunks per K-tile row
  static constexpr int VCH = DV / 8;                 // 16-byte chunks per V-tile row
  static constexpr int K_BYTES = BN * DQK * 2;
  static constexpr int V_BYTES = BN * DV * 2;
  static constexpr int STAGE_BYTES = K_BYTES + V_BYTES;
  static constexpr int LDS_BYTES = NS * STAGE_BYTES;
  // Direct-load instructions per wave per tile (each moves 64 lanes x 16 bytes).
  static constexpr int K_LOADS = BN * KCH / 64 / NWAVES;
  static constexpr int V_LOADS = BN * VCH / 64 / NWAVES;
  static constexpr int LOADS = K_LOADS + V_LOADS;
  static_assert(DQK % 32 == 0 && DV % 64 == 0, "head dims: d_qk multiple of 32, d_v multiple of 64");
  static_assert(BN % 32 == 0, "key tile must be a multiple of 32");
  static_assert((BN * KCH) % (64 * NWAVES) == 0 && (BN * VCH) % (64 * NWAVES) == 0, "tile split over waves");
  static_assert(NS >= 2 && NS <= 4 && LOADS * (NS - 1) < 64, "ring depth");
  static_assert(LDS_BYTES <= 163840, "LDS budget");
};

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
    __builtin_amdgcn_global_load_lds((global_cvoid*)(src + (size_t)key * (CH * 8) + lch * 8),
                                     (lds_void*)(stage + blk * 1024), 16, 0, 0);
  }
}

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
};

template <class C>
__global__ __attribute__((amdgpu_flat_work_group_size(C::NT, C::NT), amdgpu_waves_per_eu(C::WPE, C::WPE)))
void fa_fwd_kernel(FwdParams p) {
  using A = Attn<C>;
  constexpr int DQK = C::DQK, DV = C::DV, BN = C::BN, QB = C::QB, NS = C::NS;

  __shared__ __attribute__((aligned(1024))) unsigned char smem[C::LDS_BYTES];
  auto stage_k = [&](int s) { return smem + s * C::STAGE_BYTES; };
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

  // Start the first NS-1 tiles, then load Q while they are in flight.
  for (int t = 0; t < NS - 1 && t < nt; ++t) {
    issue_tile<C::NWAVES, BN, C::KCH>(kh, t * BN, p.sk, stage_k(t), wave, lane, kswz);
    issue_tile<C::NWAVES, BN, C::VCH>(vh, t * BN, p.sk, stage_v(t), wave, lane, vswz);
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
#define FA_NWAVES 8
#endif
#ifndef FA_QB
#define FA_QB 1
#endif
#ifndef FA_WPE
#define FA_WPE 2
#endif
#ifndef FA_NS
#define FA_NS 4
#endif

template <int DQK, int DV, bool CAUSAL>
struct Instance {
  using C = Cfg<DQK, DV, FA_BN, FA_NWAVES, FA_QB, FA_WPE, FA_NS, CAUSAL>;
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
