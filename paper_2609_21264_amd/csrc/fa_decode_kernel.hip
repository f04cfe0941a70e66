// Decode-shaped attention forward for gfx950: few query rows per key/value head (Sq * Hq / Hkv, best
// at most 32) against a long key sequence, split over workgroups by key range (the paper's
// tile-to-tile level, Alg. 2) with the log-sum-exp merge of split mode.
//
// The prefill kernel computes 256-row query blocks; a decode step has one to a few rows per query
// head, so nearly all of that work would be padding, and the shape is bound by streaming K and V from
// HBM, not by the MFMA rate. Here the Hq / Hkv query heads of one key/value head and their Sq rows are
// packed into the columns of 32-column MFMA blocks (column c = member * Sq + row; one block when
// (Hq / Hkv) * Sq <= 32), so K and V are read once per key/value head and column block, and the work
// per key is one 32-column block:
//  * A workgroup (4 waves) takes one key range ("part") of one column block of one (batch, key/value
//    head). Key tiles of 128 rows go HBM -> LDS through direct-to-LDS loads in a two-slot ring; wave w
//    loads and handles keys 32w .. 32w + 31 of each tile, so the waves run their rings without
//    barriers, and each issues tile j+1 before waiting for tile j (two tiles in flight).
//  * Per wave and tile: S^T = K Q^T (v_mfma_f32_32x32x16_bf16, Q resident as the B operand, K rows
//    in the permuted order perm32), the mask, the exact tile maximum of every column, the rescale of
//    the running sum and of O, P = 2^(s - m) rounded to bf16 in place as the B operand of
//    O^T += V^T P^T (V read with ds_read_b64_tr_b16).
//  * The waves' (m, l, O) are combined through LDS (log-sum-exp weights) and the workgroup writes
//    its part's O, normalised by the part's own sum, and the part's LSE; the merge kernel of split mode
//    combines the parts.
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

#include "fa_device.h"
#include "fa_internal.h"

namespace fa {
namespace {

#ifndef FA_DEC_WAVES
#define FA_DEC_WAVES 4
#endif
#ifndef FA_DEC_SLOTS
#define FA_DEC_SLOTS 2
#endif
constexpr int kDecWaves = FA_DEC_WAVES;   // waves per workgroup, 32 keys of each tile per wave
constexpr int kDecKeys = kDecWaves * 32;  // keys per tile
constexpr int kDecSlots = FA_DEC_SLOTS;   // ring slots: tile j + kDecSlots - 1 is loaded from step j on

template <int DQK, int DV>
struct DecCfg {
  static constexpr int KS = DQK / 16;                  // k-steps of the score product
  static constexpr int DB = DV / 32;                   // 32-dim blocks of the output
  static constexpr int KCH = DQK / 8, VCH = DV / 8;    // 16-byte chunks per K / V row
  static constexpr int K_BYTES = kDecKeys * DQK * 2;
  static constexpr int V_BYTES = kDecKeys * DV * 2;
  static constexpr int SLOT = K_BYTES + V_BYTES;
  static constexpr int LDS_BYTES = kDecSlots * SLOT;
  static constexpr int K_LOADS = kDecKeys * KCH / 64 / kDecWaves;  // direct-to-LDS loads per wave per tile
  static constexpr int V_LOADS = kDecKeys * VCH / 64 / kDecWaves;
  // Cross-wave combination: every wave's O^T as [32 columns][DV + 4] fp32 (the 16-byte pad puts
  // consecutive columns 4 banks apart), then the columns' maxima and sums.
  static constexpr int OROW = DV + 4;
  static constexpr int O_BYTES = kDecWaves * 32 * OROW * 4;
  static_assert(O_BYTES + 2 * kDecWaves * 32 * 4 <= LDS_BYTES, "combination buffers fit in the ring");
  static_assert(LDS_BYTES <= 163840, "LDS budget");
  static_assert(V_LOADS + (kDecSlots - 1) * (K_LOADS + V_LOADS) < 64 && kDecSlots >= 2, "vmcnt range");
  // Wave w's share of each tile's loads is exactly its own 32 K and V rows, so the waves never read
  // each other's LDS data in the loop (no barrier there).
  static_assert(K_LOADS * 64 == 32 * KCH && V_LOADS * 64 == 32 * VCH, "wave-private tile rows");
};

template <int DQK, int DV>
__global__ __attribute__((amdgpu_flat_work_group_size(kDecWaves * 64, kDecWaves * 64)))
void fa_decode_kernel(DecodeParams p) {
  using C = DecCfg<DQK, DV>;
  constexpr int KS = C::KS, DB = C::DB;
  __shared__ __attribute__((aligned(1024))) unsigned char smem[C::LDS_BYTES];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int i32 = lane & 31, h = lane >> 5;
  const int part = blockIdx.x % p.n_parts;
  const int cb = (blockIdx.x / p.n_parts) % p.n_cb;    // column block
  const int bg = blockIdx.x / p.n_parts / p.n_cb;      // b * Hkv + g
  const int b = bg / p.hkv, g = bg % p.hkv;
  const int c0 = cb * 32;                               // first column of the block

  // Column of this lane: query head g * group + member, row i. Padding columns (c >= rows) repeat
  // the last real column and are never stored.
  const int c = min(c0 + i32, p.rows - 1);
  const int member = c / p.sq, qi = c % p.sq;
  const int head = g * p.group + member;
  const int64_t qrow = ((int64_t)b * p.hq + head) * p.sq + qi;  // row of Q, O_part, LSE_part
  // Keys visible to the column: key j <= qi + Sk - Sq (causal), j < Sk.
  const int last_key = p.causal ? min(p.sk - 1, qi + p.sk - p.sq) : p.sk - 1;

  // Tiles [t0, t0 + nt) of this part.
  const int t0 = min(p.n_tiles, part * p.per);
  const int nt = min(p.n_tiles, t0 + p.per) - t0;
  const int k_end = min(p.sk, (t0 + nt) * kDecKeys);  // keys past this load as zeros

  bf16x8 qf[KS];
  const uint16_t* qp = p.q + qrow * DQK + 8 * h;
#pragma unroll
  for (int ks = 0; ks < KS; ++ks) qf[ks] = *reinterpret_cast<const bf16x8*>(qp + 16 * ks);

  const uint16_t* kh = p.k + (int64_t)bg * p.sk * DQK;
  const uint16_t* vh = p.v + (int64_t)bg * p.sk * DV;
  TileLoader<kDecWaves, kDecKeys, C::KCH> kload;
  TileLoader<kDecWaves, kDecKeys, C::VCH> vload;
  kload.init(kh, k_end, wave, lane, [](int r) { return k_swizzle<DQK>(r); });
  vload.init(vh, k_end, wave, lane, [](int r) { return v_swizzle<DV>(r); });
  auto kslot = [&](int t) { return smem + (t % kDecSlots) * C::SLOT; };
  auto vslot = [&](int t) { return smem + (t % kDecSlots) * C::SLOT + C::K_BYTES; };
  // Lane constants of the V transpose read (as in the prefill kernel).
  const int v_key = 8 * (lane >> 5) + ((lane & 15) >> 2);
  const int v_t = (2 * ((lane >> 4) & 1) + ((lane & 3) >> 1)) ^ v_swizzle<DV>(v_key);
  const int v_half = (lane & 1) * 8;

  f32x16 oacc[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) oacc[db] = f32x16{};
  float m_run = -INFINITY, l_run = 0.f;

  // Each wave loads and reads only its own rows of every tile (see DecCfg), so it runs its ring on
  // its own: the loads of tiles 0 .. D-1 (D = slots - 1) first, then at the start of step j those of
  // tile j+D into the slot of tile j-1, which this wave has finished reading. Step j then waits for
  // K(j) (issued after it: V(j) and the D tiles after j) before the scores and for V(j) before P V.
  constexpr int D = kDecSlots - 1;
  constexpr int L = C::K_LOADS + C::V_LOADS;
#pragma unroll
  for (int t = 0; t < D; ++t) {
    kload.issue((t0 + t) * kDecKeys, kslot(t), wave);
    vload.issue((t0 + t) * kDecKeys, vslot(t), wave);
  }
  for (int j = 0; j < nt; ++j) {
    compiler_fence();
    kload.issue((t0 + j + D) * kDecKeys, kslot(j + D), wave);
    vload.issue((t0 + j + D) * kDecKeys, vslot(j + D), wave);
    compiler_fence();
    wait_vmcnt<C::V_LOADS + D * L>();
    compiler_fence();
    const unsigned char* sK = kslot(j);
    const unsigned char* sV = vslot(j);
    const int n0 = (t0 + j) * kDecKeys + 32 * wave;  // first key of this wave's block

    // Scores: register r holds key n0 + 16 (r / 8) + 8 h + r % 8 of column i32.
    f32x16 s;
    const unsigned char* krow = sK + (32 * wave + perm32(i32)) * (DQK * 2);
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
      const u32x4 a = *reinterpret_cast<const u32x4*>(krow + (((2 * ks + h) ^ k_lane_swizzle<DQK>(i32)) << 4));
      s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bit_cast<bf16x8>(a), qf[ks], ks == 0 ? f32x16{} : s, 0, 0, 0);
    }
    // Mask keys past the column's last visible key; scale into the log2 domain.
    const int lim = last_key - n0 - 8 * h;
    float mt = -INFINITY;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const float x = (16 * (r >> 3) + (r & 7)) > lim ? -INFINITY : s[r] * p.cs;
      s[r] = x;
      mt = fmaxf(mt, x);
    }
    mt = half_swap_max(mt);
    const float m_new = fmaxf(m_run, mt);
    const float mref = m_new == -INFINITY ? 0.f : m_new;
    const float alpha = __builtin_amdgcn_exp2f(m_run - mref);  // 0 while nothing was visible
    m_run = m_new;
    float rs = 0.f;
    uint32_t pk[8];
#pragma unroll
    for (int t = 0; t < 8; ++t) {
      const float e0 = __builtin_amdgcn_exp2f(s[2 * t] - mref), e1 = __builtin_amdgcn_exp2f(s[2 * t + 1] - mref);
      rs += e0 + e1;
      pk[t] = pack_bf16x2(e0, e1);
    }
    l_run = l_run * alpha + rs;
#pragma unroll
    for (int db = 0; db < DB; ++db) oacc[db] *= alpha;
    compiler_fence();
    wait_vmcnt<D * L>();  // V(j)
    compiler_fence();
    // O^T += V^T P^T over the wave's 32 keys in two 16-key k-steps; P of keys 16 ps + 8 h .. +7 is
    // registers 8 ps .. 8 ps + 7.
#pragma unroll
    for (int ps = 0; ps < 2; ++ps) {
      const bf16x8 pb = bit_cast<bf16x8>(u32x4{pk[4 * ps], pk[4 * ps + 1], pk[4 * ps + 2], pk[4 * ps + 3]});
#pragma unroll
      for (int db = 0; db < DB; ++db) {
        const unsigned char* base = sV + (32 * wave + 16 * ps + v_key) * (DV * 2) + (((db * 4) ^ v_t) << 4) + v_half;
        const i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(base));
        const i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_i16x4*)(base + 4 * DV * 2));
        const bf16x8 va = bit_cast<bf16x8>(__builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
        oacc[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(va, pb, oacc[db], 0, 0, 0);
      }
    }
  }

  // Combine the waves: each writes its O^T, maximum and half-lane sums to LDS (no load may still be
  // writing the ring, and every wave must be done with its last tile).
  compiler_fence();
  wait_vmcnt<0>();
  compiler_fence();
  __syncthreads();
  float* ob = reinterpret_cast<float*>(smem);                 // [wave][column][OROW]
  float* mb = reinterpret_cast<float*>(smem + C::O_BYTES);    // [wave][column]
  float* lb = mb + kDecWaves * 32;                            // [wave][column]
  const float l_tot = half_swap_sum(l_run);
  if (h == 0) {
    mb[wave * 32 + i32] = m_run;
    lb[wave * 32 + i32] = l_tot;
  }
  // Register 4 g + e of oacc[db] holds dim 32 db + 8 g + 4 h + e of column i32.
  float* orow = ob + (wave * 32 + i32) * C::OROW + 4 * h;
#pragma unroll
  for (int db = 0; db < DB; ++db)
#pragma unroll
    for (int g4 = 0; g4 < 4; ++g4)
      *reinterpret_cast<f32x4*>(orow + 32 * db + 8 * g4) =
          f32x4{oacc[db][4 * g4], oacc[db][4 * g4 + 1], oacc[db][4 * g4 + 2], oacc[db][4 * g4 + 3]};
  __syncthreads();

  // Each thread finishes DV / TPC dims of one column: TPC threads per column, 32 columns.
  constexpr int TPC = kDecWaves * 64 / 32;
  const int col = tid / TPC, d0 = (tid % TPC) * (DV / TPC);
  if (c0 + col < p.rows) {
    float mw[kDecWaves], M = -INFINITY;
#pragma unroll
    for (int w = 0; w < kDecWaves; ++w) {
      mw[w] = mb[w * 32 + col];
      M = fmaxf(M, mw[w]);
    }
    float wt[kDecWaves], L = 0.f;
#pragma unroll
    for (int w = 0; w < kDecWaves; ++w) {
      wt[w] = mw[w] == -INFINITY ? 0.f : __builtin_amdgcn_exp2f(mw[w] - M);
      L += wt[w] * lb[w * 32 + col];
    }
    const float inv = L > 0.f ? 1.f / L : 0.f;
    const int cm = (c0 + col) / p.sq, ci = (c0 + col) % p.sq;
    const int64_t orow_g = ((int64_t)b * p.hq + g * p.group + cm) * p.sq + ci;
    float* dst = p.o_part + ((int64_t)part * p.total_rows + orow_g) * DV + d0;
#pragma unroll
    for (int d = 0; d < DV / TPC; d += 4) {
      f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int w = 0; w < kDecWaves; ++w)
        acc += wt[w] * *reinterpret_cast<const f32x4*>(ob + (w * 32 + col) * C::OROW + d0 + d);
      *reinterpret_cast<f32x4*>(dst + d) = acc * inv;
    }
    if (tid % TPC == 0)
      p.lse_part[(int64_t)part * p.total_rows + orow_g] = L > 0.f ? (M + log2f(L)) * 0.69314718055994530942f : -INFINITY;
  }
}

template <int DQK, int DV>
hipError_t launch_decode_instance(const DecodeParams& p, hipStream_t stream) {
  DecodeParams a = p;
  void* args[] = {&a};
  return hipLaunchKernel(reinterpret_cast<const void*>(&fa_decode_kernel<DQK, DV>),
                         dim3((unsigned)(p.batch * p.hkv * p.n_cb * p.n_parts)), dim3(kDecWaves * 64), args, 0,
                         stream);
}

}  // namespace

int decode_tile_keys() { return kDecKeys; }

hipError_t launch_decode(DecodeParams p, int d_qk, int d_v, hipStream_t stream) {
  p.n_tiles = (p.sk + kDecKeys - 1) / kDecKeys;
  p.per = (p.n_tiles + p.n_parts - 1) / p.n_parts;
  p.total_rows = (int64_t)p.batch * p.hq * p.sq;
  p.n_cb = (p.rows + 31) / 32;
  hipError_t e;
  if (d_qk == 64 && d_v == 64)
    e = launch_decode_instance<64, 64>(p, stream);
  else if (d_qk == 128 && d_v == 128)
    e = launch_decode_instance<128, 128>(p, stream);
  else if (d_qk == 192 && d_v == 128)
    e = launch_decode_instance<192, 128>(p, stream);
  else
    return hipErrorInvalidValue;
  if (e != hipSuccess) return e;
  MergeParams m;
  m.o_part = p.o_part;
  m.lse_part = p.lse_part;
  m.o = p.o;
  m.lse = p.lse;
  m.rows = p.total_rows;
  m.n_split = p.n_parts;
  return launch_merge(m, d_v, stream);
}

}  // namespace fa
