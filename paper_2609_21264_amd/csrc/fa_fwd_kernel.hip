// Fused attention forward for gfx950 (MI355X): one kernel computes, per (batch, query heads, block of
// query rows), O = softmax(scale * Q K^T) V with the online softmax of the paper's per-tile algorithm
// (Alg. 1, Sec. 2.1): key/value rows are streamed in tiles, each query row keeps a reference maximum
// and a running sum, and the unnormalised output accumulator is rescaled when the reference moves.
// Scores and probabilities live only in registers; K and V tiles are staged in LDS.
//
// Mapping onto CDNA4:
//  * A workgroup has NWAVES = 4 wavefronts (one per SIMD) sharing one key/value head; each wave owns
//    32*QB = 64 query rows of one query head: 256 rows of one head, or 128 rows of 2 heads or 64 rows
//    of 4 heads of the same GQA group when the group size allows (long instance; the short instance
//    has 32-row waves and two workgroups per CU, and the key-halves instance two sets of two 32-row
//    waves that split every key tile between them, with two or three workgroups per CU).
//  * Scores are computed transposed, S^T = K Q^T, with v_mfma_f32_32x32x16_bf16: the K tile (LDS)
//    is the A operand and the wave's Q rows (AGPRs, loaded once) are the B operand. In the 32x32
//    accumulator a lane then holds ONE query row (column = lane % 32) and 16 keys, so row
//    reductions are in-lane plus one exchange between the two lane halves (v_permlane32_swap).
//  * The A-operand rows of K are loaded in a permuted key order (bits 2 and 3 of the row index
//    swapped), which makes each 8-register group of the accumulator hold 8 consecutive keys. After
//    rounding to bf16, those registers are already the B operand of the second product
//    O^T += V^T P^T, so P never moves between lanes or through LDS.
//  * V^T is the A operand of that product and needs keys contiguous per lane. V tiles stay
//    row-major in LDS and are read with ds_read_b64_tr_b16: within each 16-lane group the
//    instruction gathers a 4 (keys) x 16 (dims) block and hands lane i the 4 keys of dim i.
//  * Three-stage software pipeline: step j runs the score MFMAs of key tile j+1, the exponentials
//    of tile j and the P V MFMAs of tile j-1. The three are independent inside a step, so the
//    softmax arithmetic is spread evenly between the MFMAs and one wave per SIMD keeps the matrix
//    unit fed while it issues VALU work (VALU work from the same wave overlaps a running MFMA).
//  * K/V tiles move HBM -> LDS with buffer loads that write LDS directly (no VGPR staging, no LDS
//    write instructions), in two rings: K tiles (2 slots by default, step j loads K(j+2)) and V
//    tiles (4 slots, step j loads V(j+2)). One wait on the wave's own loads plus one barrier per step
//    publishes the tiles of the step and frees the slots of the previous one. Rows past Sk load as
//    zeros (buffer range check), so partial tiles need no special path.
//  * 16-byte LDS chunks are XOR-swizzled per row (K: by the reading lane's key slot; V: by the key
//    mod 4) so that the lanes the LDS serves in one cycle hit 16 different bank slots. The swizzle
//    is produced by choosing each lane's source offset, since the load writes LDS lane-linearly.
//  * The output accumulators O and the Q operand live in AGPRs for the whole kernel; scores,
//    probabilities and LDS fragments use VGPRs.
//  * Causal masking skips key tiles above the diagonal entirely and applies the element mask only on
//    diagonal and tail tiles.
//  * Workgroup order: heaviest query blocks first when causal, and the workgroups that share a
//    key/value head at one query block are dispatched consecutively onto the same XCD (workgroup IDs
//    are assigned to the 8 XCDs round-robin), so their K/V tiles are served from one L2.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "fa_device.h"
#include "fa_internal.h"

namespace fa {
namespace {

constexpr float kLn2 = 0.69314718055994530942f;
// A tile's exponentials are accepted when every lane's sum of them is at most 2^8: then no
// probability exceeds 2^8 relative to the reference maximum.
constexpr float kOverflowSum = 256.0f;

// Layout of the output tile staged in LDS for coalesced stores: row R of a wave's tile (DV bf16,
// 16-byte chunks) keeps logical chunk c at chunk c ^ o_swizzle(R), with the chunk's two 8-byte
// halves exchanged when o_half(R) = 1. The accumulator layout writes 8 bytes per lane for 32 rows at
// once and the coalesced read takes 8 bytes per lane across consecutive rows; with this layout both
// touch 32 different 8-byte bank slots per cycle.
template <int DV>
__device__ __forceinline__ int o_swizzle(int r) { return DV >= 128 ? (r & 15) : ((r >> 1) & 7); }
template <int DV>
__device__ __forceinline__ int o_half(int r) { return DV >= 128 ? ((r ^ (r >> 4)) & 1) : (((r >> 1) ^ (r >> 4)) & 1); }

// The P V product is issued through inline asm so that its accumulators O stay in AGPRs for the
// whole kernel (the score product uses the builtin; its accumulators are VGPRs). The compiler does
// not model hazards of inline asm, so:
//  * mfma_out starts with s_nop 1: its P operand may have just been written by VALU, which needs
//    2 wait states before an MFMA reads it (mfma_out_settled omits them where P is old);
//  * agpr_fence() separates asm MFMA writes of O from compiler-generated accesses (initialisation,
//    rescale, epilogue) in both directions: 18 wait states cover the MFMA write-to-read distance,
//    and the operand tie keeps the order;
//  * consecutive MFMAs accumulating into exactly the same registers need no wait states.
// AG selects where O and Q live: AGPRs (one wave per SIMD, where the VGPRs alone cannot hold the
// step's scores, probabilities and fragments next to them) or VGPRs (two waves per SIMD: the
// compiler splits a wave's 256 registers evenly between the two files as soon as any AGPR is used,
// which would leave 128 VGPRs for the step; with no AGPR all 256 are VGPRs).
template <bool AG>
__device__ __forceinline__ void mfma_out(f32x16& acc, const bf16x8& v, const bf16x8& pt) {
  if constexpr (AG)
    asm("s_nop 1\n\tv_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+a"(acc) : "v"(v), "v"(pt));
  else
    asm("s_nop 1\n\tv_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+v"(acc) : "v"(v), "v"(pt));
}
// Same without the leading wait states, for operands no VALU instruction has written recently: in
// the pipelined step, P was packed a whole step earlier and V comes from LDS.
template <bool AG>
__device__ __forceinline__ void mfma_out_settled(f32x16& acc, const bf16x8& v, const bf16x8& pt) {
  if constexpr (AG)
    asm("v_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+a"(acc) : "v"(v), "v"(pt));
  else
    asm("v_mfma_f32_32x32x16_bf16 %0, %1, %2, %0" : "+v"(acc) : "v"(v), "v"(pt));
}
template <bool AG>
__device__ __forceinline__ void agpr_fence(f32x16& acc) {
  if constexpr (AG)
    asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 3" : "+a"(acc));
  else
    asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 3" : "+v"(acc));
}
// 16 bytes of Q straight into its register tuple (only read as an MFMA operand, so it never needs a
// copy). The load is not waited for here: the caller waits on vmcnt and then passes the value
// through q_ready(), which keeps every read of it after that wait.
template <bool AG>
__device__ __forceinline__ void load_q(bf16x8& r, const void* ptr) {
  if constexpr (AG)
    asm volatile("global_load_dwordx4 %0, %1, off" : "=a"(r) : "v"(ptr) : "memory");
  else
    asm volatile("global_load_dwordx4 %0, %1, off" : "=v"(r) : "v"(ptr) : "memory");
}
template <bool AG>
__device__ __forceinline__ void q_ready(bf16x8& r) {
  if constexpr (AG)
    asm volatile("" : "+a"(r));
  else
    asm volatile("" : "+v"(r));
}

// Compile-time configuration of one kernel instance: head dimensions, key-tile width, waves per
// workgroup, 32-row query blocks per wave, causal masking, split mode, workgroups sharing a CU (OCC),
// K and V fragments read ahead from LDS (KPF, VPF), K and V ring slots in LDS (NKR, NVR), and the
// parts each key tile is split into between the waves (KSPLIT).
template <int DQK_, int DV_, int BN_, int NWAVES_, int QB_, bool CAUSAL_, bool SPLIT_, int OCC_, int KPF_, int VPF_,
          int NKR_, int NVR_, int KSPLIT_ = 1>
struct Cfg {
  static constexpr int DQK = DQK_, DV = DV_, BN = BN_, NWAVES = NWAVES_, QB = QB_;
  // KSPLIT = 2: the waves form two sets of NWAVES / 2 (RWAVES) that own the same query rows; set k
  // takes the k-th 32-key half of every key tile (WBN keys per wave and tile), and the two partial
  // results of each row are merged in LDS at the end.
  static constexpr int KSPLIT = KSPLIT_, RWAVES = NWAVES / KSPLIT_, WBN = BN_ / KSPLIT_;
  static constexpr int KPF = KPF_, VPF = VPF_;
  static constexpr int OCC = OCC_;  // workgroups sharing a CU
  static constexpr bool CAUSAL = CAUSAL_;
  // SPLIT: each workgroup takes one of n_split contiguous parts of its query block's key tiles and
  // writes a partial result (O normalised by its own row sum, fp32, and its LSE) for a merge pass.
  static constexpr bool SPLIT = SPLIT_;
  static constexpr int NT = NWAVES * 64;
  // Waves per SIMD the registers are budgeted for: the workgroup's own (4 SIMDs per CU) times the
  // workgroups that share a CU (OCC_).
  static constexpr int WPE = (NWAVES > 4 ? NWAVES / 4 : 1) * OCC_;
  static constexpr int BM = RWAVES * 32 * QB;  // query rows per workgroup holding one query head
  static constexpr int KCH = DQK / 8;          // 16-byte chunks per K-tile row
  static constexpr int VCH = DV / 8;           // 16-byte chunks per V-tile row
  static constexpr int K_BYTES = BN * DQK * 2;
  static constexpr int V_BYTES = BN * DV * 2;
  // Ring slots. Step j loads K(j + KA) into the slot of K(j) and V(j + VA) into the slot of V(j-2):
  // both were last read in step j-1, which every wave has finished at the barrier of step j.
  static constexpr int NKR = NKR_, NVR = NVR_;
  static constexpr int KA = NKR, VA = NVR - 2;  // how far ahead step j loads K and V tiles
  static constexpr int LDS_BYTES = NKR * K_BYTES + NVR * V_BYTES;
  // Direct-to-LDS loads per wave per tile (each moves 64 lanes x 16 bytes).
  static constexpr int K_LOADS = BN * KCH / 64 / NWAVES;
  static constexpr int V_LOADS = BN * VCH / 64 / NWAVES;
  static_assert(DQK % 32 == 0 && DV % 64 == 0, "head dims: d_qk multiple of 32, d_v multiple of 64");
  static_assert(BN % 64 == 0, "key tiles of whole 64-key units");
  static_assert((BN * KCH) % (64 * NWAVES) == 0 && (BN * VCH) % (64 * NWAVES) == 0, "tile split over waves");
  // KA - 1 <= VA <= KA: V(j-1) is issued before K(j+1) (so one counted wait covers both), and the
  // prologue's groups j = -KA .. -1 hold every tile's first load.
  static_assert(NKR >= 2 && NKR + 1 <= NVR && NVR <= NKR + 2, "ring sizes");
  static_assert(KA * (K_LOADS + V_LOADS) < 64 && VA * (K_LOADS + V_LOADS) < 64, "vmcnt range");
  static_assert(LDS_BYTES * OCC_ <= 163840, "LDS budget of the workgroups sharing a CU");
  static_assert(KSPLIT == 1 || (KSPLIT == 2 && !SPLIT && NWAVES % 2 == 0), "key halves: two wave sets, not split mode");
};

// Division by a divisor that is fixed for the launch, as a multiply-high and two shifts (Granlund and
// Montgomery, "Division by invariant integers using multiplication", PLDI 1994, the algorithm for
// unsigned 32-bit operands): with l = ceil(log2 d) and m = floor(2^32 (2^l - d) / d) + 1, every 32-bit
// n has n / d = (t + ((n - t) >> min(l, 1))) >> max(l - 1, 0), t = mulhi(m, n). The host computes m and
// the two shifts (6 bits: min(l, 1) | max(l - 1, 0) << 1); the kernel's work decomposition then needs
// no division sequence (a runtime division by a value the compiler cannot see is ~25 instructions).
struct FastDiv {
  uint32_t m, sh;
};
FastDiv make_fastdiv(uint32_t d) {
  uint32_t l = 0;
  while ((uint64_t{1} << l) < d) ++l;
  const uint64_t m = ((uint64_t{1} << 32) * ((uint64_t{1} << l) - d)) / d + 1;
  return {static_cast<uint32_t>(m), (l < 1 ? l : 1u) | ((l > 0 ? l - 1 : 0u) << 1)};
}
__device__ __forceinline__ uint32_t fast_div(uint32_t n, uint32_t m, uint32_t sh) {
  const uint32_t t = __umulhi(m, n);
  return (t + ((n - t) >> (sh & 1u))) >> (sh >> 1);
}

// What the work decomposition needs, all uniform over the launch: workgroups per query block of one
// key/value head (`group`: the GQA group size over the query heads a workgroup packs), key/value heads,
// batch, query blocks per head, the items in whole XCD spans (below), and the fast divisions by
// `group`, the key/value heads and the batch (their shifts packed 6 bits apart in bits 0-17; bits
// 18-19 hold log2 of the query heads packed per workgroup).
struct WorkMap {
  int group, hkv, batch, n_qtiles, full;
  uint32_t m_group, m_hkv, m_batch, shifts;
};

// Map a hardware workgroup index to (batch, key/value head, member, query block); the member selects
// which of the key/value head's query heads the workgroup takes. Workgroup t runs on XCD t % 8.
// Logical work items are ordered heaviest query block first (causal), then batch, key/value head and
// member; each group of `group` consecutive items (the workgroups of one key/value head at one query
// block) is placed on one XCD, and groups go to XCDs round-robin (`full` = the items in whole spans of
// 8 groups; the rest keep their order). FAST divides through
// the multiply-high constants, else with the compiler's division sequence (the long instance: there
// the faster prologue measured no gain in time, and on the 128K workload it shifted the relative
// start times of the workgroups that stream one K/V head through an XCD's L2 enough to double the L2
// misses; the mapping is the same either way).
template <bool FAST>
__device__ __forceinline__ void decode_workgroup(uint32_t t, const WorkMap& w, bool causal, int& b, int& kvh,
                                                 int& member, int& qtile) {
  if constexpr (FAST) {
    const uint32_t G = w.group, sg = w.shifts & 63u, sh = (w.shifts >> 6) & 63u, sb = (w.shifts >> 12) & 63u;
    uint32_t L = t;
    if (t < (uint32_t)w.full) {
      const uint32_t xcd = t % kNumXcd, slot = t / kNumXcd, sq = fast_div(slot, w.m_group, sg);
      L = (sq * kNumXcd + xcd) * G + (slot - sq * G);
    }
    const uint32_t r = fast_div(L, w.m_group, sg);
    member = (int)(L - r * G);
    const uint32_t r2 = fast_div(r, w.m_hkv, sh);
    kvh = (int)(r - r2 * (uint32_t)w.hkv);
    const uint32_t qt = fast_div(r2, w.m_batch, sb);
    b = (int)(r2 - qt * (uint32_t)w.batch);
    qtile = causal ? w.n_qtiles - 1 - (int)qt : (int)qt;
  } else {
    const int G = w.group;
    int L = (int)t;
    if (L < w.full) {
      const int xcd = L % kNumXcd, slot = L / kNumXcd;
      L = ((slot / G) * kNumXcd + xcd) * G + slot % G;
    }
    member = L % G;
    int r = L / G;
    kvh = r % w.hkv;
    r /= w.hkv;
    b = r % w.batch;
    const int qt = r / w.batch;
    qtile = causal ? w.n_qtiles - 1 - qt : qt;
  }
}

// Per-wave state and the math of the pipelined step.
//
// Reference maximum (the lazy form of Alg. 1's running maximum): the first tile sets m_run to the
// exact row maximum. Afterwards the per-element maximum is not computed: each lane's sum of its
// tile exponentials bounds every one of them, so when all lane sums stay <= 2^8 no probability
// exceeds 2^8 and the tile is final. Otherwise (a new maximum well above the reference; rare) the
// tile is redone from its exact row maximum, with O and l rescaled by 2^(m_old - m_new) (rebase).
// O / l is invariant under the choice of reference, and l >= 1 since the reference is always a
// score that has been seen.
template <class C>
struct Attn {
  static constexpr int DQK = C::DQK, DV = C::DV, BN = C::WBN, QB = C::QB;  // BN: this wave's keys of a tile
  static constexpr int KS = DQK / 16;  // k-steps of the score product
  static constexpr int KB = BN / 32;   // 32-key blocks per tile
  static constexpr int DB = DV / 32;   // 32-dim blocks of the output
  static constexpr int PS = BN / 16;   // k-steps of the P V product (16-key chunks)

  typedef f32x16 Scores[KB][QB];    // S^T of one tile, raw (unscaled)
  typedef uint32_t Probs[KB][QB][8];  // P of one tile as packed bf16 pairs

  static constexpr int NMS = KS * KB * QB;  // score MFMAs per tile
  static constexpr int NMP = PS * DB * QB;  // P V MFMAs per tile
  static constexpr int NSL = NMS + NMP;     // MFMA slots per step
  static constexpr bool AG = C::WPE == 1;   // O and Q in AGPRs
  static constexpr int NEP = KB * QB * 8;   // exponential pairs per lane per tile
  static constexpr int NVF = PS * DB;       // V fragments per tile
  static constexpr int KPF = C::KPF;        // K fragments read ahead
  static constexpr int VPF = C::VPF;        // V fragments read ahead

  int i32, h, qw, diag, sk;
  const uint16_t* kg;  // this workgroup's K head in global memory (rebase only)
  float cs;            // scale * log2(e), signed
  float mask_val;      // a score that cs maps to -inf
  int v_key, v_t, v_half;
  bf16x8 qf[QB][KS];
  f32x16 oacc[DB][QB];
  float m_run[QB], l_run[QB];

  // Slot order of a step: the P V MFMAs of tile j-1 first (chunk c of P, 16 keys, in slots
  // [c * E0, (c + 1) * E0)), then the score MFMAs of tile j+1 (32-key-block-major, so that the score
  // accumulators of block kb of the new tile are written only after the exponentials of block kb of
  // the current one, and the two score tiles overlap in registers only partly).
  static constexpr int E0 = NMP / PS;
  static constexpr bool slot_is_score(int sl) { return sl >= NMP; }

  __device__ __forceinline__ u32x4 kfrag(const unsigned char* sK, int ks, int kb) const {
    const int row = kb * 32 + perm32(i32);
    return *reinterpret_cast<const u32x4*>(sK + row * (DQK * 2) + (((ks * 2 + h) ^ k_lane_swizzle<DQK>(i32)) << 4));
  }
  // A operand V^T[dims db*32 + 0..31][keys 16*ps + 0..15]: lane (group G, slot j) points the
  // transpose read at key 16*ps + 8*(G/2) + j/4 (then +4), dims db*32 + 16*(G%2) + 4*(j%4).
  __device__ __forceinline__ bf16x8 vfrag(const unsigned char* sV, int ps, int db) const {
    const unsigned char* base = sV + (ps * 16 + v_key) * (DV * 2) + (((db * 4) ^ v_t) << 4) + v_half;
    const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(base));
    const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(base + 4 * DV * 2));
    return bit_cast<bf16x8>(__builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
  }

  // Score MFMA number i of a tile in 32-key-block-major order (kb, ks, qb); K fragments (sequence
  // f = kb*KS + ks) are read KPF ahead.
  __device__ __forceinline__ void score_mfma(Scores& s, u32x4 (&kf)[KB * KS], const unsigned char* sK, int i) {
    const int kb = i / (KS * QB), ks = (i / QB) % KS, qb = i % QB, f = kb * KS + ks;
    if (qb == 0 && f + KPF < KB * KS) kf[f + KPF] = kfrag(sK, (f + KPF) % KS, (f + KPF) / KS);
    s[kb][qb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bit_cast<bf16x8>(kf[f]), qf[qb][ks],
                                                        ks == 0 ? f32x16{} : s[kb][qb], 0, 0, 0);
  }
  __device__ __forceinline__ void scores(Scores& s, const unsigned char* sK) {
    u32x4 kf[KB * KS];
#pragma unroll
    for (int f = 0; f < KPF && f < KB * KS; ++f) kf[f] = kfrag(sK, f % KS, f / KS);
#pragma unroll
    for (int i = 0; i < NMS; ++i) score_mfma(s, kf, sK, i);
  }

  // Masked keys of tile n0 (key > i + diag, or key >= Sk) get mask_val. The select is a bit
  // select on the sign of (lim - key offset): a compare per element would need a scalar register
  // pair per mask, and the scheduler hoists all 64 of them.
  __device__ __forceinline__ void mask_tile(Scores& s, int n0) const {
    const uint32_t mv = __float_as_uint(mask_val);
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      const int row = qw + qb * 32 + i32;
      const int last_key = C::CAUSAL ? min(row + diag, sk - 1) : sk - 1;
      const int lim = last_key - n0 - 8 * h;  // key offset kb*32 + 16*(r/8) + r%8 is masked iff > lim
#pragma unroll
      for (int kb = 0; kb < KB; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const uint32_t m = (uint32_t)((lim - (kb * 32 + 16 * (r >> 3) + (r & 7))) >> 31);  // all ones if masked
          s[kb][qb][r] = __uint_as_float((__float_as_uint(s[kb][qb][r]) & ~m) | (mv & m));
        }
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

  // Element schedule of the step: the NEL = 2 * NEP exponentials of a tile are spread
  // one by one over the NSL MFMA slots (element e in slot e * NSL / NEL), each as one fma and one
  // exp2 right after the slot's MFMA; the two adds and the pack of pair u follow in the slot after
  // the one of its second element. At d = 128 a slot then carries 3 and 6 full-rate-equivalent VALU
  // instructions in turn, within what a 32-cycle MFMA absorbs. A pair's pack writes P chunk c only
  // after the P V MFMAs of chunk c (slots [c * E0, (c + 1) * E0)) for every c >= 1, so the old and new
  // P share registers there; chunk 0 is written earlier and takes registers of its own.
  static constexpr int NEL = 2 * NEP;
  static constexpr int elem_begin(int sl) { return (sl * NEL + NSL - 1) / NSL; }
  static constexpr int elem_end(int sl) { return ((sl + 1) * NEL + NSL - 1) / NSL; }
  static constexpr bool packs_follow_pv() {
    for (int u = 0; u < NEP; ++u) {
      int sl = 0;
      while (elem_end(sl) <= 2 * u + 1) ++sl;  // slot of element 2u+1
      const int c = u / (QB * 4);             // P chunk (16 keys) of pair u
      if (c >= 1 && sl + 1 < (c + 1) * E0) return false;
    }
    return true;
  }
  static_assert(packs_follow_pv(), "a pack would overwrite P of a chunk before its P V MFMAs");
  static constexpr bool at_most_two_elems_per_slot() {
    for (int sl = 0; sl < NSL; ++sl)
      if (elem_end(sl) - elem_begin(sl) > 2) return false;
    return true;
  }

  // Element e of a tile: p = 2^(cs * s - m_ref).
  __device__ __forceinline__ float exp_elem(int e, const Scores& cur, const float (&mref)[QB]) const {
    const int u = e >> 1, qb = u % QB, rp = (u / QB) % 8, kb = u / (QB * 8);
    float x = __builtin_amdgcn_exp2f(fmaf(cur[kb][qb][2 * rp + (e & 1)], cs, -mref[qb]));
    asm volatile("" : "+v"(x));
    return x;
  }
  // Pair u: the lane's row sum and the bf16 pair. The first pair of each row block starts the sum.
  __device__ __forceinline__ void pack_pair(int u, float e0, float e1, Probs& pk, float (&rs)[QB]) const {
    const int qb = u % QB, rp = (u / QB) % 8, kb = u / (QB * 8);
    if (u < QB)
      rs[qb] = e0 + e1;
    else
      rs[qb] += e0 + e1;
    pk[kb][qb][rp] = pack_bf16x2(e0, e1);
    asm volatile("" : "+v"(pk[kb][qb][rp]));
  }

  // P V MFMA number p of a tile (order ps, db, qb), V fragments read VPF ahead. `settled`: P was
  // written long before (in the step: one step earlier), so no wait states are needed.
  __device__ __forceinline__ void pv_mfma(int p, const Probs& pk, bf16x8 (&vf)[NVF], const unsigned char* sV,
                                          bool settled = false) {
    const int t = p / QB, qb = p % QB, ps = t / DB, db = t % DB;
    if (qb == 0 && t + VPF < NVF) vf[t + VPF] = vfrag(sV, (t + VPF) / DB, (t + VPF) % DB);
    const int kb = ps >> 1, base = (ps & 1) * 4;
    const u32x4 w = {pk[kb][qb][base], pk[kb][qb][base + 1], pk[kb][qb][base + 2], pk[kb][qb][base + 3]};
    if (settled)
      mfma_out_settled<AG>(oacc[db][qb], vf[t], bit_cast<bf16x8>(w));
    else
      mfma_out<AG>(oacc[db][qb], vf[t], bit_cast<bf16x8>(w));
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
  // tile's scores are recomputed from K in global memory (rows clamped to Sk-1, masked anyway): by
  // the end of the step the raw scores are gone and the tile's LDS slot holds a later tile.
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
        agpr_fence<AG>(oacc[db][qb]);
        oacc[db][qb] *= alpha;
        agpr_fence<AG>(oacc[db][qb]);
      }
      mref[qb] = m_new == -INFINITY ? 0.f : m_new;
    }
#pragma unroll
    for (int u = 0; u < NEP; ++u) {
      const float e0 = exp_elem(2 * u, cur, mref), e1 = exp_elem(2 * u + 1, cur, mref);
      pack_pair(u, e0, e1, pk, rs);
    }
  }

  // One pipeline step: P V of tile j-1 (pk_old, V slot sVo), exponentials of tile j (cur, key n0,
  // into pk_new) and scores of tile j+1 (K slot sKn, into nxt).
  // `issue(k)` starts load k (0 <= k < LOADS) of the tiles this step prefetches; the loads are spread
  // one every NSL / LOADS slots, between MFMAs (a burst of them would stall the wave).
  template <class Issue>
  __device__ __forceinline__ void step(Scores& cur, Scores& nxt, Probs& pk_new, const Probs& pk_old,
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
    static_assert(at_most_two_elems_per_slot(), "ev holds the elements of two slots");
    float ev[4];  // exponentials in flight, element e in ev[e % 4]
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int sl = 0; sl < NSL; ++sl) {
      {
        constexpr int NLD = C::K_LOADS + C::V_LOADS, SP = NSL / NLD;
        static_assert(SP >= 1, "more loads than slots");
        if (sl % SP == SP / 2 && sl / SP < NLD) issue(sl / SP);
      }
      if (slot_is_score(sl))
        score_mfma(nxt, kf, sKn, sl - NMP);
      else
        pv_mfma(sl, pk_old, vf, sVo, true);
      __builtin_amdgcn_sched_barrier(0);  // the slot's MFMA is issued before its VALU work
      if (sl > 0) {
#pragma unroll
        for (int e = elem_begin(sl - 1); e < elem_end(sl - 1); ++e)
          if (e & 1) pack_pair(e >> 1, ev[(e - 1) % 4], ev[e % 4], pk_new, rs);
      }
#pragma unroll
      for (int e = elem_begin(sl); e < elem_end(sl); ++e) ev[e % 4] = exp_elem(e, cur, mref);
      __builtin_amdgcn_sched_barrier(0);
    }
#pragma unroll
    for (int e = elem_begin(NSL - 1); e < elem_end(NSL - 1); ++e)
      if (e & 1) pack_pair(e >> 1, ev[(e - 1) % 4], ev[e % 4], pk_new, rs);
    bool over = false;
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) over = over || !(rs[qb] <= kOverflowSum);
    if (__builtin_amdgcn_ballot_w64(over) != 0) rebase(pk_new, rs, n0, masked);
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) l_run[qb] += rs[qb];
  }
};

// The kernel body, shared by the two entry kernels below.
template <class C>
__device__ __forceinline__ void fa_fwd_body(FwdParams p, const WorkMap wm) {
  using A = Attn<C>;
  constexpr int DQK = C::DQK, DV = C::DV, BN = C::BN, QB = C::QB;

  __shared__ __attribute__((aligned(1024))) unsigned char smem[C::LDS_BYTES];
  auto kswz = [](int row) { return k_swizzle<DQK>(row); };
  auto vswz = [](int row) { return v_swizzle<DV>(row); };

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  A st;
  st.i32 = lane & 31;
  st.h = lane >> 5;
  // Lane constants of the V transpose read: group G = lane/16, slot j = lane%16.
  st.v_key = 8 * (lane >> 5) + ((lane & 15) >> 2);                             // key in the 16-key step
  st.v_t = (2 * ((lane >> 4) & 1) + ((lane & 3) >> 1)) ^ v_swizzle<DV>(st.v_key);  // low chunk bits, swizzled
  st.v_half = (lane & 1) * 8;                                                  // byte offset in the chunk
  st.sk = p.sk;

  // Split mode: workgroup t takes part t / n_wg of work item t % n_wg.
  const int split = C::SPLIT ? (int)(blockIdx.x / p.n_wg) : 0;
  int b, g, member, qtile;
  decode_workgroup<(C::OCC > 1)>(C::SPLIT ? blockIdx.x % (uint32_t)p.n_wg : blockIdx.x, wm, C::CAUSAL, b, g, member,
                                 qtile);
  // Query heads packed per workgroup (HW = 1, 2 or 4, the largest that divides the GQA group size):
  // the waves split into HW heads of the same key/value head, each taking NWAVES / HW consecutive
  // 32*QB-row chunks of the block's rows, so that all heads of the workgroup share every K/V tile
  // and, when HW = NWAVES, every wave visits the same key tiles (no wave idles through the tiles of
  // a causal diagonal that its rows do not see).
  // With key halves (KSPLIT = 2) the same applies within each wave set: wave w belongs to set
  // w / RWAVES, which takes keys [kpart, kpart + WBN) of every tile, and to row chunk w % RWAVES.
  const int hw_log = (int)((wm.shifts >> 18) & 3u);
  const int kset = C::KSPLIT > 1 ? wave / C::RWAVES : 0, rwave = C::KSPLIT > 1 ? wave % C::RWAVES : wave;
  const int kpart = kset * C::WBN;                       // first key of this wave's part of a tile
  const int rw = C::RWAVES >> hw_log;                    // row chunks per head
  const int bmr = rw * 32 * QB;                          // query rows of the block
  const int hq = g * p.group + (member << hw_log) + rwave / rw;
  const uint16_t* __restrict__ qh = p.q + (size_t)(b * p.hq + hq) * p.sq * DQK;

  const int q0 = qtile * bmr;
  st.qw = q0 + (rwave % rw) * 32 * QB;  // first query row of this wave
  st.diag = p.sk - p.sq;        // key j is visible to query i iff j <= i + diag

  // Key tiles this workgroup visits, and how many leading ones need no mask for any of its rows.
  int kv_end = p.sk;
  int n_plain = p.sk / BN;
  if (C::CAUSAL) {
    const int last_row = min(q0 + bmr, p.sq) - 1;
    kv_end = max(0, min(p.sk, last_row + st.diag + 1));
    n_plain = min(n_plain, max(0, q0 + st.diag + 1) / BN);
  }
  // Key tiles [t0, t0 + nt) of the query block: all of them, or one contiguous part in split mode.
  int t0 = 0, nt = (kv_end + BN - 1) / BN;
  if (C::SPLIT) {
    const int per = (nt + p.n_split - 1) / p.n_split;
    t0 = min(nt, split * per);
    nt = min(nt, t0 + per) - t0;
  }
  const int kb0 = t0 * BN;                     // first key of the range
  n_plain = min(max(n_plain - t0, 0), nt);     // leading tiles of the range that need no mask
  const int kv_lim = min(kv_end, kb0 + nt * BN);  // keys loaded; past it the tile loads read zeros

  // Q rows of this wave as B operands of the score product, resident in AGPRs: lane (i32, h) holds
  // row qw+32*qb+i32, dims 16*ks + 8*h .. +7. Rows past Sq read row Sq-1 instead; their outputs are
  // never stored. Issued first, waited for together with the first K tile below.
#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    const int row = min(st.qw + qb * 32 + st.i32, p.sq - 1);
#pragma unroll
    for (int ks = 0; ks < A::KS; ++ks) load_q<A::AG>(st.qf[qb][ks], qh + (size_t)row * DQK + ks * 16 + st.h * 8);
  }
  // What comes from the argument block (not preloaded) is used only from here on.
  const uint16_t* __restrict__ kh = p.k + (size_t)(b * p.hkv + g) * p.sk * DQK;
  const uint16_t* __restrict__ vh = p.v + (size_t)(b * p.hkv + g) * p.sk * DV;
  st.kg = kh;
  st.cs = p.cs;
  st.mask_val = p.cs < 0.f ? INFINITY : -INFINITY;

  // Rings: step j loads K(j+KA) and V(j+VA) (the group of step j); the prologue loads the groups of
  // j = -KA .. -1 (with the defaults KA = VA = 2: K0, V0, K1, V1 in this order), each group's V tile
  // only from V0 on. Every group is issued in full: a tile at or past the last one loads
  // zeros into a slot nobody reads any more, so the number of loads issued after any given one is a
  // constant and every wait below is a fixed count.
  TileLoader<C::NWAVES, BN, C::KCH> kload;
  TileLoader<C::NWAVES, BN, C::VCH> vload;
  kload.init(kh, kv_lim, wave, lane, kswz);
  vload.init(vh, kv_lim, wave, lane, vswz);
  // (tile indices are never negative: unsigned remainders, a mask for the power-of-two ring sizes)
  auto kslot = [&](int t) { return smem + ((unsigned)t % C::NKR) * C::K_BYTES; };
  auto vslot = [&](int t) { return smem + C::NKR * C::K_BYTES + ((unsigned)t % C::NVR) * C::V_BYTES; };
  // This wave's keys of tile t (rows kpart .. kpart + WBN - 1 of the slot). The K and V swizzles
  // repeat every 32 rows, so a part starting at row 32 reads like a tile of its own.
  auto kmine = [&](int t) { return kslot(t) + kpart * (DQK * 2); };
  auto vmine = [&](int t) { return vslot(t) + kpart * (DV * 2); };
#pragma unroll
  for (int g = -C::KA; g < 0; ++g) {
    kload.issue(kb0 + (g + C::KA) * BN, kslot(g + C::KA), wave);
    if (g + C::VA >= 0) vload.issue(kb0 + (g + C::VA) * BN, vslot(g + C::VA), wave);
  }
  // Q and K0 must have landed: issued after K0 are V0 when VA = KA, then the groups of j = -KA+1 ..
  // -1 (K and V each, since VA >= KA - 1).
  wait_vmcnt<(C::VA == C::KA ? C::V_LOADS : 0) + (C::KA - 1) * (C::K_LOADS + C::V_LOADS)>();
#pragma unroll
  for (int qb = 0; qb < QB; ++qb)
#pragma unroll
    for (int ks = 0; ks < A::KS; ++ks) q_ready<A::AG>(st.qf[qb][ks]);

#pragma unroll
  for (int qb = 0; qb < QB; ++qb) {
    st.m_run[qb] = -INFINITY;
    st.l_run[qb] = 0.f;
#pragma unroll
    for (int db = 0; db < A::DB; ++db) {
      st.oacc[db][qb] = f32x16{};
      agpr_fence<A::AG>(st.oacc[db][qb]);
    }
  }

  typename A::Scores sA, sB;
  typename A::Probs pA, pB;
  if (nt > 0) {
    // Tile 0: scores, mask, exact row maxima. P of "tile -1" is zero; its P V step reads the K1
    // slot, which has landed (or holds zeros) and is not written during step 0: finite data times
    // zero adds nothing.
    compiler_fence();
    __builtin_amdgcn_s_barrier();
    compiler_fence();
    st.scores(sA, kmine(0));
    if (n_plain == 0) st.mask_tile(sA, kb0 + kpart);
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) st.m_run[qb] = st.row_max(sA, qb);
#pragma unroll
    for (int kb = 0; kb < A::KB; ++kb)
#pragma unroll
      for (int qb = 0; qb < QB; ++qb)
#pragma unroll
        for (int r = 0; r < 8; ++r) pB[kb][qb][r] = 0u;
  }
  // Before step j: K(j+1) and V(j-1) must have landed. K(j+1) belongs to the group of step j+1-KA;
  // this wave's loads issued after it are that group's V tile and the KA-2 groups after it (with
  // the defaults only V(j+1)); V(j-1), from the group of step j+1-NVR, came before it.
  // The barrier then publishes every wave's part and guarantees that all waves are done with step
  // j-1, whose slots (K(j), V(j-2)) the loads of step j overwrite.
  // The steps run in order j = 0, 1, ..., so the buffers of the tiles a step loads are the previous
  // step's moved on by one tile (they start one tile before those of step 0).
  int krem, vrem;
  u32x4 gk = kload.rsrc_walk(kb0 + (C::KA - 1) * BN, krem), gv = vload.rsrc_walk(kb0 + (C::VA - 1) * BN, vrem);
  uint32_t gkl = 0, gvl = 0;
  auto sync_step = [&](int j) {
    wait_vmcnt<C::V_LOADS + (C::KA - 2) * (C::K_LOADS + C::V_LOADS)>();
    compiler_fence();
    __builtin_amdgcn_s_barrier();
    compiler_fence();
    kload.advance(gk, krem);
    gkl = kload.lds(kslot(j + C::KA), wave);
    vload.advance(gv, vrem);
    gvl = vload.lds(vslot(j + C::VA), wave);
  };
  auto issue = [&](int k) {
    if (k < C::K_LOADS)
      kload.issue_one(gk, gkl, k);
    else
      vload.issue_one(gv, gvl, k - C::K_LOADS);
  };
  // Steps in pairs so that the two score tiles and the two P tiles swap roles without copies. A step
  // masks its current tile from tile n_plain on; tile 0 was masked above when n_plain = 0, and masking
  // it again in step 0 changes nothing (masked scores already hold mask_val), so the test needs no
  // j > 0 term (one scalar compare per step instead of two compares and the mask logic).
  int j = 0;
  for (; j + 1 < nt; j += 2) {
    sync_step(j);
    st.step(sA, sB, pA, pB, kmine(j + 1), j > 0 ? vmine(j - 1) : kmine(1), j >= n_plain,
            kb0 + j * BN + kpart, issue);
    sync_step(j + 1);
    st.step(sB, sA, pB, pA, kmine(j + 2), vmine(j), j + 1 >= n_plain, kb0 + (j + 1) * BN + kpart, issue);
  }
  if (j < nt) {
    sync_step(j);
    st.step(sA, sB, pA, pB, kmine(j + 1), j > 0 ? vmine(j - 1) : kmine(1), j >= n_plain,
            kb0 + j * BN + kpart, issue);
  }
  if (nt > 0) {
    // P V of the last tile, on a selected copy of P: two calls would leave O in different
    // registers and the copies that merge them could read MFMA results before they are written.
    // (The select is a bit mask: a ternary on the elements would be folded into a select of the
    // two arrays' addresses, which forces both into scratch memory.) V(nt-1) belongs to the load
    // group of step nt-1-VA; the VA groups after it may still be in flight.
    wait_vmcnt<C::VA * (C::K_LOADS + C::V_LOADS)>();
    compiler_fence();
    __builtin_amdgcn_s_barrier();
    compiler_fence();
    typename A::Probs pl;
    const uint32_t take_a = (nt & 1) ? 0xffffffffu : 0u;
#pragma unroll
    for (int kb = 0; kb < A::KB; ++kb)
#pragma unroll
      for (int qb = 0; qb < QB; ++qb)
#pragma unroll
        for (int r = 0; r < 8; ++r) pl[kb][qb][r] = (pA[kb][qb][r] & take_a) | (pB[kb][qb][r] & ~take_a);
    st.pv_tile(pl, vmine(nt - 1));
  }

  // No load may still be writing this workgroup's LDS when it exits (the prologue issues loads even
  // when there is no key tile to visit), and the output tile is staged in the ring slots below: every
  // wave's loads must have landed and every wave must be done with the last V tile.
  wait_vmcnt<0>();
  compiler_fence();
  __builtin_amdgcn_s_barrier();
  compiler_fence();

  if constexpr (C::KSPLIT > 1) {
    // Merge of the two key halves (the combination step of Alg. 2 inside the workgroup): the second
    // wave set hands its O, reference maxima and lane row sums to the wave of the first set with the
    // same rows through LDS, lane by lane (both hold the same rows and dims in the same registers),
    // and exits. With m = max(m_a, m_b): O = O_a 2^(m_a - m) + O_b 2^(m_b - m), likewise l; a half
    // that saw no visible key (m = -inf, O = 0, l = 0) gets weight 0. The exchange area lies past
    // the first set's output staging tiles.
    constexpr int NF = A::DB * QB * 16;  // O floats per lane
    constexpr int XCH_OFF = C::RWAVES * 32 * QB * DV * 2;
    static_assert(XCH_OFF + C::RWAVES * (NF + 2 * QB) * 64 * 4 <= C::LDS_BYTES, "exchange area fits the LDS");
    float* xch = reinterpret_cast<float*>(smem + XCH_OFF) + rwave * (NF + 2 * QB) * 64;
    if (kset == 1) {
#pragma unroll
      for (int qb = 0; qb < QB; ++qb) {
#pragma unroll
        for (int db = 0; db < A::DB; ++db) {
          agpr_fence<A::AG>(st.oacc[db][qb]);
#pragma unroll
          for (int g4 = 0; g4 < 4; ++g4) {
            const f32x16& o = st.oacc[db][qb];
            *reinterpret_cast<f32x4*>(xch + (((qb * A::DB + db) * 4 + g4) * 64 + lane) * 4) =
                f32x4{o[4 * g4], o[4 * g4 + 1], o[4 * g4 + 2], o[4 * g4 + 3]};
          }
        }
        xch[NF * 64 + qb * 64 + lane] = st.m_run[qb];
        xch[NF * 64 + (QB + qb) * 64 + lane] = st.l_run[qb];
      }
    }
    compiler_fence();
    __builtin_amdgcn_s_barrier();
    compiler_fence();
    if (kset == 1) return;
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      const float m_b = xch[NF * 64 + qb * 64 + lane], l_b = xch[NF * 64 + (QB + qb) * 64 + lane];
      const float m_a = st.m_run[qb], m = fmaxf(m_a, m_b);
      const float wa = m_a == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m_a - m);
      const float wb = m_b == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(m_b - m);
      st.m_run[qb] = m;
      st.l_run[qb] = st.l_run[qb] * wa + l_b * wb;
#pragma unroll
      for (int db = 0; db < A::DB; ++db) {
        agpr_fence<A::AG>(st.oacc[db][qb]);
#pragma unroll
        for (int g4 = 0; g4 < 4; ++g4) {
          const f32x4 ob = *reinterpret_cast<const f32x4*>(xch + (((qb * A::DB + db) * 4 + g4) * 64 + lane) * 4);
#pragma unroll
          for (int e = 0; e < 4; ++e) st.oacc[db][qb][4 * g4 + e] = st.oacc[db][qb][4 * g4 + e] * wa + ob[e] * wb;
        }
      }
    }
  }

  // ---- epilogue: O = acc / l, LSE = ln 2 * (m + log2 l) ---------------------------------------
  if constexpr (C::SPLIT) {
    // Partial result of this part of the key range, for the merge pass: O normalised by this part's
    // row sum (fp32, 16 bytes per lane and block) and this part's LSE; an empty part gives O = 0 and
    // LSE = -inf, which the merge weighs with 0.
#pragma unroll
    for (int qb = 0; qb < QB; ++qb)
#pragma unroll
      for (int db = 0; db < A::DB; ++db) agpr_fence<A::AG>(st.oacc[db][qb]);
    const size_t head_rows = ((size_t)split * p.batch * p.hq + (size_t)b * p.hq + hq) * p.sq;
#pragma unroll
    for (int qb = 0; qb < QB; ++qb) {
      const float l_tot = half_swap_sum(st.l_run[qb]);
      const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
      const int row = st.qw + qb * 32 + st.i32;
      if (row < p.sq) {
        float* orow = p.o_part + (head_rows + row) * DV;
#pragma unroll
        for (int db = 0; db < A::DB; ++db)
#pragma unroll
          for (int g4 = 0; g4 < 4; ++g4)
            *reinterpret_cast<f32x4*>(orow + db * 32 + 8 * g4 + 4 * st.h) =
                f32x4{st.oacc[db][qb][4 * g4] * inv, st.oacc[db][qb][4 * g4 + 1] * inv,
                      st.oacc[db][qb][4 * g4 + 2] * inv, st.oacc[db][qb][4 * g4 + 3] * inv};
        if (st.h == 0) p.lse_part[head_rows + row] = l_tot > 0.f ? (st.m_run[qb] + log2f(l_tot)) * kLn2 : -INFINITY;
      }
    }
  } else {
    // O goes through LDS so that each store instruction writes whole rows (1 KiB contiguous); stored
    // straight from the accumulator layout, every instruction would touch 32 rows 16 bytes at a time.
    constexpr int RB = DV * 2;           // bytes per output row
    constexpr int WROWS = 32 * QB;       // rows per wave
    static_assert(C::NWAVES * WROWS * RB <= C::LDS_BYTES, "output staging fits in the ring slots");
    unsigned char* stage = smem + wave * WROWS * RB;
  #pragma unroll
    for (int qb = 0; qb < QB; ++qb)
  #pragma unroll
      for (int db = 0; db < A::DB; ++db) agpr_fence<A::AG>(st.oacc[db][qb]);
    {
      const int osw = o_swizzle<DV>(st.i32) << 4;             // qb * 32 leaves the low 5 row bits alone
      const int ohalf = (st.h ^ o_half<DV>(st.i32)) << 3;
  #pragma unroll
      for (int qb = 0; qb < QB; ++qb) {
        const float l_tot = half_swap_sum(st.l_run[qb]);
        const float inv = l_tot > 0.f ? 1.f / l_tot : 0.f;
        unsigned char* srow = stage + (qb * 32 + st.i32) * RB + ohalf;
  #pragma unroll
        for (int db = 0; db < A::DB; ++db)
  #pragma unroll
          for (int g4 = 0; g4 < 4; ++g4) {
            const int c = 4 * db + g4;  // 16-byte chunk: dims 8c .. 8c+7, this lane's half 4h .. 4h+3
            const uint32_t w0 = pack_bf16x2(st.oacc[db][qb][4 * g4] * inv, st.oacc[db][qb][4 * g4 + 1] * inv);
            const uint32_t w1 = pack_bf16x2(st.oacc[db][qb][4 * g4 + 2] * inv, st.oacc[db][qb][4 * g4 + 3] * inv);
            *reinterpret_cast<uint2*>(srow + ((c << 4) ^ osw)) = make_uint2(w0, w1);
          }
        const int row = st.qw + qb * 32 + st.i32;
        if (p.lse != nullptr && st.h == 0 && row < p.sq)
          p.lse[(size_t)(b * p.hq + hq) * p.sq + row] =
              l_tot > 0.f ? (st.m_run[qb] + log2f(l_tot)) * kLn2 : -INFINITY;
      }
    }
    // Each wave reads back only its own rows, so no barrier: LDS serves one wave's accesses in order.
    {
      constexpr int CPR = RB / 16;        // 16-byte chunks per row
      constexpr int RPI = 64 / CPR;       // rows per store instruction
      const int c = lane % CPR;
      uint16_t* ohead = p.o + (size_t)(b * p.hq + hq) * p.sq * DV;
      // All reads first, pinned before the stores as a group: the compiler would otherwise sink each
      // read into its store's row guard and wait out an LDS round trip per store.
      constexpr int NIT = WROWS / RPI;
      u32x4 ov[NIT];
  #pragma unroll
      for (int it = 0; it < NIT; ++it) {
        const int r = it * RPI + lane / CPR;
        const unsigned char* chunk = stage + r * RB + ((c ^ o_swizzle<DV>(r)) << 4);
        const int hl = o_half<DV>(r) << 3;
        const uint2 x = *reinterpret_cast<const uint2*>(chunk + hl);
        const uint2 y = *reinterpret_cast<const uint2*>(chunk + (hl ^ 8));
        ov[it] = u32x4{x.x, x.y, y.x, y.y};
      }
  #pragma unroll
      for (int it = 0; it < NIT; ++it) asm volatile("" : "+v"(ov[it]));
  #pragma unroll
      for (int it = 0; it < NIT; ++it) {
        const int row = st.qw + it * RPI + lane / CPR;
        if (row < p.sq) *reinterpret_cast<u32x4*>(ohead + (size_t)row * DV + c * 8) = ov[it];
      }
    }
  }
}

// Entry kernels. The long instance reads everything from the argument block. The instances with
// several workgroups per CU (short and key halves), whose workgroups are short chains on which the
// first loads' latency is felt, take the values their prologue needs first as leading scalar
// arguments, which the command processor preloads into SGPRs before the first instruction
// (kernel-argument preloading, enabled at build time for the first 14 SGPRs of a kernel's leading
// scalar arguments), and issue their Q loads before they read the argument block. Preloading is kept
// off the long instance: it slows the launch of each wave, and on the 128K
// workload the spread-out starts of the workgroups that stream one K/V head through an XCD's L2
// doubled the L2 misses, at no gain in time.
template <class C>
__global__ __attribute__((amdgpu_flat_work_group_size(C::NT, C::NT), amdgpu_waves_per_eu(C::WPE, C::WPE)))
void fa_fwd_kernel(FwdParams p) {
  fa_fwd_body<C>(p, WorkMap{p.group >> ((p.shifts >> 18) & 3u), p.hkv, p.batch, p.n_qtiles, p.full, p.m_group, p.m_hkv,
                            p.m_batch, p.shifts});
}
template <class C>
__global__ __attribute__((amdgpu_flat_work_group_size(C::NT, C::NT), amdgpu_waves_per_eu(C::WPE, C::WPE)))
void fa_fwd_kernel_preload(const uint16_t* a_q, int a_sq, int a_sk, int a_hq, int a_batch, int a_hkv, int a_group,
                           int a_nqt, int a_full, uint32_t a_mg, uint32_t a_mh, uint32_t a_mb, uint32_t a_shifts,
                           FwdParams p) {
  p.q = a_q;
  p.sq = a_sq;
  p.sk = a_sk;
  p.hq = a_hq;
  p.batch = a_batch;
  p.hkv = a_hkv;
  p.group = a_group;
  p.n_qtiles = a_nqt;
  fa_fwd_body<C>(p, WorkMap{a_group >> ((a_shifts >> 18) & 3u), a_hkv, a_batch, a_nqt, a_full, a_mg, a_mh, a_mb,
                            a_shifts});
}

// The instances. Long: 4 waves x 64 query rows (256 row-heads per workgroup), one workgroup per CU,
// one wave per SIMD; the register budget of a wave (O 128 + Q 64 AGPRs at d = 128, two score tiles
// and P in VGPRs) is what fixes 64 query rows per wave. K tiles are loaded two ahead: a third K slot
// measured 2-3 % slower on the 8K, 4K-d192 and 128K prefill shapes (one box, interleaved).
// Short: 4 waves x 32 query rows (128 row-heads per workgroup), two workgroups per CU (two waves per SIMD,
// 256 registers each, O and Q in VGPRs), shallower fragment prefetch at d = 128 so that the step fits
// the registers without spilling, and a V ring of 3 slots at d = 128 (so that two rings fit one CU's
// LDS) and 4 at d = 64 (V tiles loaded two steps ahead; 3-8 % faster than 3 slots on the d = 64
// shapes it runs, while a deeper K ring measured slower). It
// runs problems with few query blocks (short sequences, few heads), where 256-row blocks leave CUs
// idle and each block's serial chain of steps sets the time: on the paper's S = 512 and 2048 GPT-2
// and BERT shapes and the 128K single-head workload it measured 1.2-1.4x faster than the long
// instance, and slower once the long instance's grid fills the GPU. At d_qk = 192 two waves per SIMD
// do not fit, so those problems always run the long instance.
#ifndef FA_BN
#define FA_BN 64
#endif
#ifndef FA_NWAVES
#define FA_NWAVES 4
#endif
#ifndef FA_QB
#define FA_QB 2
#endif
#ifndef FA_KPF
#define FA_KPF 2
#endif
#ifndef FA_VPF
#define FA_VPF 6
#endif
#ifndef FA_NKR
#define FA_NKR 2
#endif
#ifndef FA_NVR
#define FA_NVR 4
#endif

template <int DQK, int DV, bool CAUSAL, bool SPLIT = false>
struct Instance {
  using C = Cfg<DQK, DV, FA_BN, FA_NWAVES, FA_QB, CAUSAL, SPLIT, 1, FA_KPF, FA_VPF, FA_NKR, FA_NVR>;
};
template <int DQK, int DV, bool CAUSAL>
struct ShortInstance {
  using C = Cfg<DQK, DV, 64, 4, 1, CAUSAL, false, 2, DQK >= 128 ? 1 : 2, DQK >= 128 ? 2 : 6, 2, DQK >= 128 ? 3 : 4>;
};
// The short instance at d = 64 with 128-key tiles, for keys of at least kWideTileKeys: a step then
// carries 32 MFMAs per wave instead of 16, over which the per-step waits, barrier, load issue and
// addressing are spread (250 VGPRs; the 16 KiB tiles allow a V ring of 3 slots, 80 KiB per
// workgroup). Measured against the 64-key tiles (one box, interleaved): 1.5-6 % faster from 1 536
// keys on (BERT-Base and -Large S2048 1.05-1.06x, GPT-2 Small S8192 and S16384 1.02-1.03x), level at
// 1 024, 1.5 % slower at 512 keys (workload 2), where the four steps of a block leave too little to
// overlap with the pipeline's fill and drain.
template <int DQK, int DV, bool CAUSAL>
struct ShortWideInstance {
  using C = Cfg<DQK, DV, 128, 4, 1, CAUSAL, false, 2, 2, 6, 2, 3>;
};
constexpr int kWideTileKeys = 1024;
// Key halves: 4 waves as two sets of 2 x 32 query rows (64 row-heads per workgroup), each set taking
// one 32-key half of every tile; three workgroups per CU at d = 64 (three waves per SIMD, 132 VGPRs,
// 48 KiB of LDS each), two at d = 128 (208 VGPRs, 80 KiB). It runs problems whose grid of long-
// instance blocks is small enough that each workgroup's chain of steps sets the time: the chain
// keeps its number of steps but each step carries half the work per wave. V fragments are read 4
// ahead at d = 64 and 2 at d = 128, the best of 2-8 measured (one box, interleaved).
template <int DQK, int DV, bool CAUSAL>
struct HalfInstance {
  using C = Cfg<DQK, DV, 64, 4, 1, CAUSAL, false, DQK >= 128 ? 2 : 3, 2, DQK >= 128 ? 2 : 4, 2, DQK >= 128 ? 3 : 4, 2>;
};

// Largest grid of long-instance blocks (256 row-heads) that runs the short instance instead. At
// d = 128 the CU count of MI355X, where the long instance would leave CUs idle. At d = 64, where a
// step carries twice the softmax work per MFMA and the long instance's one wave per SIMD exposes it,
// the short instance's two waves per SIMD pay off up to four blocks per CU: measured 5-17 % faster on
// causal and non-causal GPT-2-shaped problems of 384-768 blocks, level at 1024-1152, 3-4 % slower from
// 1536 blocks on (one box, interleaved).
constexpr int64_t kShortMaxBlocks64 = 1024, kShortMaxBlocks128 = 256;
// Largest grid of such blocks that runs the key-halves instance, by head dimension and masking.
// Causal problems have a longest chain of steps (the last query block's) that halving each step's
// work per wave shortens; problems without a mask gain only while the grid leaves SIMDs idle. At
// d = 128 causal grids of 256 blocks measured 0.96-1.06x against the short instance (the paper's
// Llama S = 2048 shapes on the slow side), so they stay with it.
constexpr int64_t kHalfMaxCausal64 = 320, kHalfMaxFull64 = 64, kHalfMaxCausal128 = 192, kHalfMaxFull128 = 128;

enum class Kind { kLong, kShort, kHalf };

Kind pick_instance(const FwdParams& p, int d_qk, int d_v, bool causal) {
  if (!((d_qk == 64 && d_v == 64) || (d_qk == 128 && d_v == 128))) return Kind::kLong;
  const int bm = Instance<64, 64, false>::C::BM;
  const int64_t blocks = (int64_t)p.batch * p.hq * ((p.sq + bm - 1) / bm);
  const int64_t half_max = d_qk == 64 ? (causal ? kHalfMaxCausal64 : kHalfMaxFull64)
                                      : (causal ? kHalfMaxCausal128 : kHalfMaxFull128);
  if (blocks <= half_max) return Kind::kHalf;
  return blocks <= (d_qk == 64 ? kShortMaxBlocks64 : kShortMaxBlocks128) ? Kind::kShort : Kind::kLong;
}

// log2 of the query heads a workgroup of `nwaves` waves packs: 4, 2 or 1 heads, the largest that
// divides the GQA group size (and the wave count).
int packed_heads_log2(int group, int nwaves) {
  if (group % 4 == 0 && nwaves % 4 == 0) return 2;
  if (group % 2 == 0 && nwaves % 2 == 0) return 1;
  return 0;
}

template <class C>
hipError_t launch_cfg(FwdParams p, hipStream_t stream) {
  const int hw_log = packed_heads_log2(p.group, C::RWAVES);
  const int gi = p.group >> hw_log;  // workgroups per key/value head and query block
  const int bmr = (C::RWAVES >> hw_log) * 32 * C::QB;
  p.n_qtiles = (p.sq + bmr - 1) / bmr;
  p.n_wg = p.batch * p.hkv * gi * p.n_qtiles;
  const int span = kNumXcd * gi;
  p.full = (p.n_wg / span) * span;
  const FastDiv fg = make_fastdiv(gi), fh = make_fastdiv(p.hkv), fb = make_fastdiv(p.batch);
  p.m_group = fg.m;
  p.m_hkv = fh.m;
  p.m_batch = fb.m;
  p.shifts = fg.sh | fh.sh << 6 | fb.sh << 12 | (uint32_t)hw_log << 18;
  const dim3 grid(p.n_wg * (C::SPLIT ? p.n_split : 1));
  if constexpr (C::OCC > 1) {
    void* args[] = {&p.q,        &p.sq,   &p.sk,      &p.hq,    &p.batch,   &p.hkv,    &p.group,
                    &p.n_qtiles, &p.full, &p.m_group, &p.m_hkv, &p.m_batch, &p.shifts, &p};
    return hipLaunchKernel(reinterpret_cast<const void*>(&fa_fwd_kernel_preload<C>), grid, dim3(C::NT), args, 0,
                           stream);
  } else {
    void* args[] = {&p};
    return hipLaunchKernel(reinterpret_cast<const void*>(&fa_fwd_kernel<C>), grid, dim3(C::NT), args, 0, stream);
  }
}

template <int DQK, int DV, bool CAUSAL, bool SPLIT>
hipError_t launch_instance(FwdParams p, Kind kind, hipStream_t stream) {
  if constexpr (!SPLIT && DQK != 192) {
    if (kind == Kind::kHalf) return launch_cfg<typename HalfInstance<DQK, DV, CAUSAL>::C>(p, stream);
  }
  if constexpr (!SPLIT && DQK != 192) {
    if (kind == Kind::kShort) {
      if constexpr (DQK == 64) {
        if (p.sk >= kWideTileKeys) return launch_cfg<typename ShortWideInstance<DQK, DV, CAUSAL>::C>(p, stream);
      }
      return launch_cfg<typename ShortInstance<DQK, DV, CAUSAL>::C>(p, stream);
    }
  }
  return launch_cfg<typename Instance<DQK, DV, CAUSAL, SPLIT>::C>(p, stream);
}

template <bool SPLIT>
hipError_t launch_dims(FwdParams p, int d_qk, int d_v, bool causal, hipStream_t stream) {
  const Kind sh = SPLIT ? Kind::kLong : pick_instance(p, d_qk, d_v, causal);
  if (d_qk == 64 && d_v == 64)
    return causal ? launch_instance<64, 64, true, SPLIT>(p, sh, stream)
                  : launch_instance<64, 64, false, SPLIT>(p, sh, stream);
  if (d_qk == 128 && d_v == 128)
    return causal ? launch_instance<128, 128, true, SPLIT>(p, sh, stream)
                  : launch_instance<128, 128, false, SPLIT>(p, sh, stream);
  if (d_qk == 192 && d_v == 128)
    return causal ? launch_instance<192, 128, true, SPLIT>(p, sh, stream)
                  : launch_instance<192, 128, false, SPLIT>(p, sh, stream);
  return hipErrorInvalidValue;
}

// Merge of the n_split partial results of every query row (log-sum-exp combination): with
// M = max_s LSE_s, w_s = exp(LSE_s - M), O = sum_s w_s O_s / sum_s w_s and LSE = M + ln(sum_s w_s).
// A row whose parts are all empty (LSE_s = -inf) gets O = 0 and LSE = -inf. A row is handled by
// DV / 4 * pg threads: thread (g, q) takes output dims 4q .. 4q+3 of the parts s = g (mod pg), so the
// loads of a row are independent and in flight together; the pg partial maxima, weighted sums and
// weight sums are combined through LDS. pg is the smallest power of two >= n_split, at most
// 256 / (DV / 4); a workgroup of 256 threads takes 256 / (DV / 4 * pg) rows. Reads fp32, writes bf16
// (round to nearest even) and the fp32 LSE.
template <int DV>
__global__ __launch_bounds__(256) void fa_merge_kernel(MergeParams p, int pg) {
  constexpr int TD = DV / 4;     // threads per part group (one per 4 output dims)
  constexpr int NG = 256 / TD;   // part groups per workgroup
  __shared__ float s_m[NG], s_den[NG];
  __shared__ f32x4 s_acc[NG][TD];
  const int q = threadIdx.x % TD, gw = threadIdx.x / TD;  // group within the workgroup
  const int g = gw % pg;                                  // part group within the row
  const int64_t row = (int64_t)blockIdx.x * (NG / pg) + gw / pg;
  const bool live = row < p.rows;
  const int g0 = gw - g;                                  // first group of this row
  float m = -INFINITY;
  if (live)
    for (int sp = g; sp < p.n_split; sp += pg) m = fmaxf(m, p.lse_part[sp * p.rows + row]);
  if (q == 0) s_m[gw] = m;
  __syncthreads();
  float M = -INFINITY;
  for (int k = 0; k < pg; ++k) M = fmaxf(M, s_m[g0 + k]);
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  float den = 0.f;
  if (live && M != -INFINITY) {
    for (int sp = g; sp < p.n_split; sp += pg) {
      const float w = expf(p.lse_part[sp * p.rows + row] - M);
      den += w;
      acc += w * *reinterpret_cast<const f32x4*>(p.o_part + (sp * p.rows + row) * DV + 4 * q);
    }
  }
  s_acc[gw][q] = acc;
  if (q == 0) s_den[gw] = den;
  __syncthreads();
  if (live && g == 0) {
    float dsum = 0.f;
    f32x4 o = {0.f, 0.f, 0.f, 0.f};
    for (int k = 0; k < pg; ++k) {
      dsum += s_den[g0 + k];
      o += s_acc[g0 + k][q];
    }
    o *= dsum > 0.f ? 1.f / dsum : 0.f;
    f32x2 lo = {o.x, o.y}, hi = {o.z, o.w};
    *reinterpret_cast<uint2*>(p.o + row * DV + 4 * q) =
        make_uint2(bit_cast<uint32_t>(__builtin_convertvector(lo, bf16x2)),
                   bit_cast<uint32_t>(__builtin_convertvector(hi, bf16x2)));
    if (q == 0 && p.lse != nullptr) p.lse[row] = dsum > 0.f ? M + logf(dsum) : -INFINITY;
  }
}

}  // namespace

int block_rows(int d_qk, int d_v, bool causal) {
  (void)causal;
  if (d_qk == 64 && d_v == 64) return Instance<64, 64, false>::C::BM;
  if (d_qk == 128 && d_v == 128) return Instance<128, 128, false>::C::BM;
  if (d_qk == 192 && d_v == 128) return Instance<192, 128, false>::C::BM;
  return 0;
}

int instance_rows(int batch, int hq, int sq, int d_qk, int d_v, bool causal) {
  const int bm = block_rows(d_qk, d_v, causal);
  if (bm == 0 || batch < 0 || hq < 0 || sq < 0) return 0;
  FwdParams p{};
  p.batch = batch;
  p.hq = hq;
  p.sq = sq;
  switch (pick_instance(p, d_qk, d_v, causal)) {
    case Kind::kHalf:
      return HalfInstance<64, 64, false>::C::BM;
    case Kind::kShort:
      return ShortInstance<64, 64, false>::C::BM;
    default:
      return bm;
  }
}

int64_t forward_workgroups(int batch, int hq, int hkv, int sq) {
  // the long instance's grid (the other instances run only grids of at most 2 048 workgroups)
  using C = Instance<64, 64, false>::C;
  const int group = hq / hkv, hw_log = packed_heads_log2(group, C::RWAVES);
  const int64_t bmr = (C::NWAVES >> hw_log) * 32 * C::QB;
  return (int64_t)batch * hkv * (group >> hw_log) * ((sq + bmr - 1) / bmr);
}

hipError_t launch_forward(FwdParams p, int d_qk, int d_v, bool causal, hipStream_t stream) {
  return launch_dims<false>(p, d_qk, d_v, causal, stream);
}

hipError_t launch_merge(MergeParams m, int d_v, hipStream_t stream) {
  const int groups = 256 / (d_v / 4);
  int pg = 1;
  while (pg < m.n_split && pg < groups) pg *= 2;
  const int64_t rows_per_wg = groups / pg;
  const dim3 grid((unsigned)((m.rows + rows_per_wg - 1) / rows_per_wg));
  void* args[] = {&m, &pg};
  const void* k = d_v == 64 ? reinterpret_cast<const void*>(&fa_merge_kernel<64>)
                            : reinterpret_cast<const void*>(&fa_merge_kernel<128>);
  return hipLaunchKernel(k, grid, dim3(256), args, 0, stream);
}

hipError_t launch_forward_split(FwdParams p, int d_qk, int d_v, bool causal, hipStream_t stream) {
  const hipError_t e = launch_dims<true>(p, d_qk, d_v, causal, stream);
  if (e != hipSuccess) return e;
  MergeParams m;
  m.o_part = p.o_part;
  m.lse_part = p.lse_part;
  m.o = p.o;
  m.lse = p.lse;
  m.rows = (int64_t)p.batch * p.hq * p.sq;
  m.n_split = p.n_split;
  return launch_merge(m, d_v, stream);
}

}  // namespace fa
