// Internal interface between the C-ABI layer (fa_api.hip) and the kernel launchers (fa_fwd_kernel.hip:
// fused forward and split mode; fa_lbl_kernel.hip: layer-by-layer operators). Not installed; callers
// use include/fa.h.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace fa {

// Arguments of one forward launch, after host-side validation.
struct FwdParams {
  const uint16_t* q;  // bf16 [B][Hq][Sq][d_qk]
  const uint16_t* k;  // bf16 [B][Hkv][Sk][d_qk]
  const uint16_t* v;  // bf16 [B][Hkv][Sk][d_v]
  uint16_t* o;        // bf16 [B][Hq][Sq][d_v]
  float* lse;         // fp32 [B][Hq][Sq] or nullptr
  int batch, hq, hkv, sq, sk;
  int group;          // Hq / Hkv
  float cs;           // scale * log2(e), magnitude at least FLT_MIN so that an infinite (masked)
                      // score stays infinite; negative when scale < 0
  int n_qtiles;       // ceil(Sq / block rows)
  int n_wg;           // work items (query blocks): batch * hq * n_qtiles
  // Work decomposition constants (host-computed): the items in whole spans of 8 groups, and the
  // multiply-high constants for dividing by group, hkv and batch, their shifts packed 6 bits apart.
  int full;
  uint32_t m_group, m_hkv, m_batch, shifts;
  // Split mode only: number of key-range parts, and the partial results, in the caller's workspace:
  // o_part fp32 [n_split][B][Hq][Sq][d_v] (O of each part normalised by its own row sum), lse_part
  // fp32 [n_split][B][Hq][Sq].
  int n_split;
  float* o_part;
  float* lse_part;
};

// Arguments of the merge pass of split mode.
struct MergeParams {
  const float* o_part;
  const float* lse_part;
  uint16_t* o;      // bf16 [rows][d_v]
  float* lse;       // fp32 [rows] or nullptr
  int64_t rows;     // B * Hq * Sq
  int n_split;
};

// Query rows per workgroup of the long kernel instance for (d_qk, d_v, causal) when a workgroup holds
// one query head (split mode, every d_qk = 192 problem, and problems with more such blocks than the
// other instances take); 0 if not compiled in.
// With a GQA group size divisible by 2 or 4 a workgroup holds as many query heads, each with half or
// a quarter of these rows.
int block_rows(int d_qk, int d_v, bool causal);
// Query rows per workgroup holding one query head of the instance the fused forward runs for this
// problem: the long instance's block_rows() (256), the short instance's 128 or the key-halves
// instance's 64; 0 for unsupported head dimensions or negative sizes.
int instance_rows(int batch, int hq, int sq, int d_qk, int d_v, bool causal);
// Workgroups of the long instance's grid (one part per query block and packed heads).
int64_t forward_workgroups(int batch, int hq, int hkv, int sq);

// Enqueue the forward kernel for (d_qk, d_v, causal) on `stream`. Requires Sq > 0, B*Hq > 0 and a
// grid that fits; fills n_qtiles / n_wg itself. Returns the launch status of the HIP runtime.
hipError_t launch_forward(FwdParams p, int d_qk, int d_v, bool causal, hipStream_t stream);

// Split mode: the forward kernel over n_split parts of every query block's key range, writing the
// partial results, then the merge pass into O / LSE, both on `stream`. Same requirements as
// launch_forward plus n_split >= 1 and the partial buffers.
hipError_t launch_forward_split(FwdParams p, int d_qk, int d_v, bool causal, hipStream_t stream);

// The merge pass alone (d_v 64 or 128), on `stream`.
hipError_t launch_merge(MergeParams m, int d_v, hipStream_t stream);

// ---- decode-shaped problems (fa_decode_kernel.hip) -----------------------------------------------
//
// The group's query heads and their Sq rows form the columns of 32-column MFMA blocks; workgroup t
// takes part t % n_parts of column block (t / n_parts) % n_cb of (batch, key/value head)
// t / (n_parts * n_cb), and the parts are
// merged by the merge pass of split mode (same partial-result layout: o_part fp32
// [n_parts][B][Hq][Sq][d_v], lse_part fp32 [n_parts][B][Hq][Sq]).
struct DecodeParams {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  uint16_t* o;
  float* lse;
  float* o_part;
  float* lse_part;
  int batch, hq, hkv, sq, sk, group, causal;
  float cs;           // scale * log2(e), as in FwdParams
  int rows;           // group * Sq (columns)
  int n_parts;
  int n_tiles, per;   // filled by launch_decode: key tiles, tiles per part
  int n_cb;           // filled by launch_decode: 32-column blocks
  int64_t total_rows; // B * Hq * Sq, filled by launch_decode
};

// Keys per tile of the decode kernel.
int decode_tile_keys();
// Enqueue the decode kernel and the merge pass on `stream`; (d_qk, d_v) in {(64,64), (128,128), (192,128)}.
hipError_t launch_decode(DecodeParams p, int d_qk, int d_v, hipStream_t stream);

// ---- layer-by-layer (unfused) operators --------------------------------------------------------
//
// A work unit is one block of kLblRows query rows of one (batch, query head); bh = b * Hq + h. A chunk
// is a rectangle of units, query heads bh0 .. bh0+nbh-1 times query blocks qb0 .. qb0+nqb-1, that is
// either whole heads (qb0 = 0, all blocks) or part of one head (nbh = 1). Row r of the chunk, i.e.
// (bh - bh0) * Sq + (qb - qb0) * kLblRows + row in block, is row r of the spill buffers S and P
// (stride ld elements). Key extents are multiples of kLblKeys: the rows of block qb use keys
// [0, lbl_extent(qb)), the visible keys of the block's last row rounded up.
constexpr int kLblRows = 128;
constexpr int kLblKeys = 64;
// Largest Sk of the layer-by-layer operators: keeps every byte offset inside one block's rows of the
// spill buffer (kLblRows * ld * 2) below 2^30.
constexpr int kLblMaxSk = 1 << 22;

struct LblParams {
  const uint16_t* q;  // bf16 [B][Hq][Sq][d_qk]
  const uint16_t* k;  // bf16 [B][Hkv][Sk][d_qk]
  const uint16_t* v;  // bf16 [B][Hkv][Sk][d_v]
  uint16_t* s;        // bf16 scores of the chunk, row stride ld
  uint16_t* p;        // bf16 probabilities of the chunk, row stride ld (may equal s)
  uint16_t* o;        // bf16 [B][Hq][Sq][d_v]
  float* lse;         // fp32 [B][Hq][Sq] or nullptr
  int batch, hq, hkv, sq, sk, group, causal;
  int ld;             // Sk rounded up to kLblKeys
  float scale;
  int bh0, nbh, qb0, nqb;
  int xgroup;         // query heads placed together on one XCD: group if the chunk is aligned to it, else 1
  int64_t rows;       // rows of the chunk
};

bool lbl_scores_supported(int d_qk);
bool lbl_pv_supported(int d_v);
// Each enqueues one kernel over the chunk on `stream` and returns the launch status.
hipError_t launch_lbl_scores(const LblParams& p, int d_qk, hipStream_t stream);
hipError_t launch_lbl_softmax(const LblParams& p, hipStream_t stream);
hipError_t launch_lbl_pv(const LblParams& p, int d_v, hipStream_t stream);

}  // namespace fa
