// Internal interface between the C-ABI layer (fa_api.hip) and the kernel launchers
// (fa_fwd_kernel.hip). Not installed; callers use include/fa.h.
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

// Query rows per workgroup of the kernel instance for (d_qk, d_v, causal); 0 if not compiled in.
int block_rows(int d_qk, int d_v, bool causal);

// Enqueue the forward kernel for (d_qk, d_v, causal) on `stream`. Requires Sq > 0, B*Hq > 0 and a
// grid that fits; fills n_qtiles / n_wg itself. Returns the launch status of the HIP runtime.
hipError_t launch_forward(FwdParams p, int d_qk, int d_v, bool causal, hipStream_t stream);

// Split mode: the forward kernel over n_split parts of every query block's key range, writing the
// partial results, then the merge pass into O / LSE, both on `stream`. Same requirements as
// launch_forward plus n_split >= 1 and the partial buffers.
hipError_t launch_forward_split(FwdParams p, int d_qk, int d_v, bool causal, hipStream_t stream);

}  // namespace fa
