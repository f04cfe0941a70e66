// C ABI of the fused attention forward (declared in include/fa.h): host-side argument checks, then
// one kernel launch on the caller's stream. No allocation, no synchronisation, no global state.
#include <float.h>
#include <limits.h>
#include <math.h>
#include <stdint.h>

#include "fa.h"
#include "fa_internal.h"

namespace {

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }

// Bytes of the split-mode workspace: partial O (fp32, d_v per row) and LSE (fp32) for every row and
// part; -1 if the count overflows.
int64_t split_workspace_bytes(int B, int Hq, int Sq, int d_v, int n_split) {
  if (B <= 0 || Hq <= 0 || Sq <= 0 || d_v <= 0 || n_split <= 0) return 0;
  const int64_t bh = static_cast<int64_t>(B) * Hq;  // < 2^62
  const int64_t per_row = (static_cast<int64_t>(d_v) + 1) * 4 * n_split;  // < 2^44
  if (bh > INT64_MAX / Sq) return -1;
  const int64_t rows = bh * Sq;
  if (rows > INT64_MAX / per_row) return -1;
  return rows * per_row;
}

fa_status_t forward(const void* Q, const void* K, const void* V, void* O, float* LSE, int B, int Hq, int Hkv,
                    int Sq, int Sk, int d_qk, int d_v, float scale, int causal, void* stream, int n_split = 0,
                    void* workspace = nullptr, size_t workspace_bytes = 0) {
  if (B < 0 || Hq < 0 || Hkv < 0 || Sq < 0 || Sk < 0) return FA_ERR_BAD_SHAPE;
  if (Hq > 0 && (Hkv <= 0 || Hq % Hkv != 0)) return FA_ERR_BAD_SHAPE;
  const int bm = fa::block_rows(d_qk, d_v, causal != 0);
  if (bm == 0) return FA_ERR_UNSUPPORTED;
  // A pointer may be NULL only when the array it addresses has no element.
  const bool q_rows = static_cast<int64_t>(B) * Hq * Sq > 0;
  const bool kv_rows = static_cast<int64_t>(B) * Hkv * Sk > 0;
  if ((q_rows && (Q == nullptr || O == nullptr)) || (kv_rows && (K == nullptr || V == nullptr)))
    return FA_ERR_NULL_POINTER;
  if (!isfinite(scale)) return FA_ERR_BAD_SCALE;
  const double c = fabs(static_cast<double>(scale)) * 1.4426950408889634074;  // |scale| * log2(e)
  if (c > FLT_MAX) return FA_ERR_BAD_SCALE;
  if (!aligned(Q, 16) || !aligned(K, 16) || !aligned(V, 16) || !aligned(O, 16)) return FA_ERR_UNSUPPORTED;
  if (!aligned(LSE, 4)) return FA_ERR_UNSUPPORTED;
  // Offsets inside one head are 32-bit in the kernel.
  const int64_t dmax = d_qk > d_v ? d_qk : d_v;
  if (static_cast<int64_t>(Sq) * dmax > INT_MAX || static_cast<int64_t>(Sk) * dmax > INT_MAX) return FA_ERR_BAD_SHAPE;
  if (B == 0 || Hq == 0 || Sq == 0) return FA_OK;
  const int64_t n_qtiles = (static_cast<int64_t>(Sq) + bm - 1) / bm;
  const int64_t n_wg = static_cast<int64_t>(B) * Hq * n_qtiles;
  if (n_wg > INT_MAX || static_cast<int64_t>(B) * Hq > INT_MAX || static_cast<int64_t>(B) * Hkv > INT_MAX)
    return FA_ERR_BAD_SHAPE;
  if (n_split > 0) {
    if (n_wg * n_split > INT_MAX) return FA_ERR_BAD_SHAPE;
    const int64_t need = split_workspace_bytes(B, Hq, Sq, d_v, n_split);
    if (need < 0 || workspace == nullptr || static_cast<uint64_t>(need) > workspace_bytes) return FA_ERR_WORKSPACE;
    if (!aligned(workspace, 16)) return FA_ERR_UNSUPPORTED;
  }

  fa::FwdParams p{};
  p.q = static_cast<const uint16_t*>(Q);
  p.k = static_cast<const uint16_t*>(K);
  p.v = static_cast<const uint16_t*>(V);
  p.o = static_cast<uint16_t*>(O);
  p.lse = LSE;
  p.batch = B;
  p.hq = Hq;
  p.hkv = Hkv;
  p.sq = Sq;
  p.sk = Sk;
  p.group = Hq / Hkv;
  const float cmag = c < FLT_MIN ? FLT_MIN : static_cast<float>(c);
  p.cs = scale < 0.f ? -cmag : cmag;
  hipError_t err;
  if (n_split > 0) {
    const int64_t rows = static_cast<int64_t>(B) * Hq * Sq;
    p.n_split = n_split;
    p.o_part = static_cast<float*>(workspace);
    p.lse_part = p.o_part + rows * n_split * d_v;
    err = fa::launch_forward_split(p, d_qk, d_v, causal != 0, static_cast<hipStream_t>(stream));
  } else {
    err = fa::launch_forward(p, d_qk, d_v, causal != 0, static_cast<hipStream_t>(stream));
  }
  return err == hipSuccess ? FA_OK : FA_ERR_HIP;
}

}  // namespace

extern "C" {

fa_status_t fa_fwd_ex(const void* Q, const void* K, const void* V, void* O, float* LSE, int B, int Hq, int Hkv,
                      int Sq, int Sk, int d_qk, int d_v, float scale, int causal, void* stream) {
  return forward(Q, K, V, O, LSE, B, Hq, Hkv, Sq, Sk, d_qk, d_v, scale, causal, stream);
}

fa_status_t fa_fwd(const void* Q, const void* K, const void* V, void* O, int B, int Hq, int Hkv, int Sq, int Sk,
                   int d, float scale, int causal, void* stream) {
  return forward(Q, K, V, O, nullptr, B, Hq, Hkv, Sq, Sk, d, d, scale, causal, stream);
}

fa_status_t fa_fwd_split(const void* Q, const void* K, const void* V, void* O, float* LSE, int B, int Hq, int Hkv,
                         int Sq, int Sk, int d_qk, int d_v, float scale, int causal, int n_split, void* workspace,
                         size_t workspace_bytes, void* stream) {
  if (n_split < 1) return FA_ERR_BAD_SHAPE;
  return forward(Q, K, V, O, LSE, B, Hq, Hkv, Sq, Sk, d_qk, d_v, scale, causal, stream, n_split, workspace,
                 workspace_bytes);
}

int fa_fwd_split_parts(int n_cu, int B, int Hq, int Sq, int Sk, int d_qk, int d_v, int causal) {
  const int bm = fa::block_rows(d_qk, d_v, causal != 0);
  if (bm == 0 || n_cu <= 0 || B <= 0 || Hq <= 0 || Sq <= 0 || Sk < 0) return 0;
  // Enough workgroups for about two per CU, but no part shorter than 8 key tiles (the fixed cost of
  // a workgroup and of the merge would dominate). The query block with the most keys sees all Sk.
  const int64_t items = static_cast<int64_t>(B) * Hq * ((static_cast<int64_t>(Sq) + bm - 1) / bm);
  const int64_t max_parts = (static_cast<int64_t>(Sk) + 64 * 8 - 1) / (64 * 8);
  int64_t parts = (2 * static_cast<int64_t>(n_cu)) / items;
  if (parts > max_parts) parts = max_parts;
  return parts < 1 ? 1 : static_cast<int>(parts);
}

size_t fa_fwd_split_workspace_bytes(int B, int Hq, int Sq, int d_v, int n_split) {
  const int64_t n = split_workspace_bytes(B, Hq, Sq, d_v, n_split);
  return n < 0 ? SIZE_MAX : static_cast<size_t>(n);
}

const char* fa_status_str(fa_status_t s) {
  switch (s) {
    case FA_OK: return "FA_OK";
    case FA_ERR_NULL_POINTER: return "FA_ERR_NULL_POINTER";
    case FA_ERR_BAD_SHAPE: return "FA_ERR_BAD_SHAPE";
    case FA_ERR_UNSUPPORTED: return "FA_ERR_UNSUPPORTED";
    case FA_ERR_BAD_SCALE: return "FA_ERR_BAD_SCALE";
    case FA_ERR_HIP: return "FA_ERR_HIP";
    case FA_ERR_WORKSPACE: return "FA_ERR_WORKSPACE";
  }
  return "unknown status";
}

int fa_block_rows(int d_qk, int d_v, int causal) { return fa::block_rows(d_qk, d_v, causal != 0); }

}  // extern "C"
