// C ABI of the attention forward (declared in include/fa.h): host-side argument checks, then kernel
// launches on the caller's stream (fused forward, split mode, decode-shaped path, layer-by-layer
// operators). No allocation and no synchronisation; the only state is the per-device address of the
// static scratch array of fa_fwd_decode_noalloc.
#include <float.h>
#include <limits.h>
#include <math.h>
#include <stdint.h>

#include <atomic>
#include <mutex>

#include "fa.h"
#include "fa_internal.h"

// Static scratch of the allocation-free decode entry point: fa_fwd_decode_noalloc keeps its partial
// results in this file-scope device array instead of a caller workspace. Every device the library
// runs on holds its own copy (allocated with the code object, kept until the process ends). On the
// host, `scratch` names a host-side stand-in, not a device address: the device address is looked up
// once per device with hipGetSymbolAddress (with that device current, scratch_for_stream below) and
// only that address is passed to kernels.
static __device__ __align__(256) unsigned char scratch[FA_NOALLOC_SCRATCH_BYTES];

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

// Checks shared by the fused entry points (fa_fwd_ex, fa_fwd_split, fa_fwd_decode and
// fa_fwd_decode_noalloc), in the order fa.h documents: sizes, head dimensions, pointers, scale,
// alignment, index ranges. On FA_OK, *cs holds scale * log2(e) as the kernels take it (magnitude at
// least FLT_MIN, so that a masked score stays infinite; negative when scale < 0).
fa_status_t check_fused(const void* Q, const void* K, const void* V, const void* O, const float* LSE, int B, int Hq,
                        int Hkv, int Sq, int Sk, int d_qk, int d_v, float scale, int causal, float* cs) {
  if (B < 0 || Hq < 0 || Hkv < 0 || Sq < 0 || Sk < 0) return FA_ERR_BAD_SHAPE;
  if (Hq > 0 && (Hkv <= 0 || Hq % Hkv != 0)) return FA_ERR_BAD_SHAPE;
  if (fa::block_rows(d_qk, d_v, causal != 0) == 0) return FA_ERR_UNSUPPORTED;
  // A pointer may be NULL only when the array it addresses has no element.
  const bool q_rows = static_cast<int64_t>(B) * Hq * Sq > 0;
  const bool kv_rows = static_cast<int64_t>(B) * Hkv * Sk > 0;
  if ((q_rows && (Q == nullptr || O == nullptr)) || (kv_rows && (K == nullptr || V == nullptr)))
    return FA_ERR_NULL_POINTER;
  if (!isfinite(scale)) return FA_ERR_BAD_SCALE;
  const double c = fabs(static_cast<double>(scale)) * 1.4426950408889634074;  // |scale| * log2(e)
  if (c > FLT_MAX) return FA_ERR_BAD_SCALE;
  if (!aligned(Q, 16) || !aligned(K, 16) || !aligned(V, 16) || !aligned(O, 16) || !aligned(LSE, 4))
    return FA_ERR_UNSUPPORTED;
  // Offsets inside one head are 32-bit in the kernels.
  const int64_t dmax = d_qk > d_v ? d_qk : d_v;
  if (static_cast<int64_t>(Sq) * dmax > INT_MAX || static_cast<int64_t>(Sk) * dmax > INT_MAX) return FA_ERR_BAD_SHAPE;
  const float cmag = c < FLT_MIN ? FLT_MIN : static_cast<float>(c);
  *cs = scale < 0.f ? -cmag : cmag;
  return FA_OK;
}

fa_status_t forward(const void* Q, const void* K, const void* V, void* O, float* LSE, int B, int Hq, int Hkv,
                    int Sq, int Sk, int d_qk, int d_v, float scale, int causal, hipStream_t stream, int n_split = 0,
                    void* workspace = nullptr, size_t workspace_bytes = 0) {
  float cs = 0.f;
  const fa_status_t st = check_fused(Q, K, V, O, LSE, B, Hq, Hkv, Sq, Sk, d_qk, d_v, scale, causal, &cs);
  if (st != FA_OK) return st;
  if (B == 0 || Hq == 0 || Sq == 0) return FA_OK;
  const int64_t n_wg = fa::forward_workgroups(B, Hq, Hkv, Sq);
  if (n_wg > INT_MAX || static_cast<int64_t>(B) * Hq > INT_MAX || static_cast<int64_t>(B) * Hkv > INT_MAX)
    return FA_ERR_BAD_SHAPE;
  if (n_split > 0) {
    if (n_wg * n_split > INT_MAX) return FA_ERR_BAD_SHAPE;
    if (static_cast<int64_t>(B) * Hq * Sq > INT_MAX) return FA_ERR_BAD_SHAPE;  // merge: a workgroup per row at most
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
  p.cs = cs;
  hipError_t err;
  if (n_split > 0) {
    const int64_t rows = static_cast<int64_t>(B) * Hq * Sq;
    p.n_split = n_split;
    p.o_part = static_cast<float*>(workspace);
    p.lse_part = p.o_part + rows * n_split * d_v;
    err = fa::launch_forward_split(p, d_qk, d_v, causal != 0, stream);
  } else {
    err = fa::launch_forward(p, d_qk, d_v, causal != 0, stream);
  }
  return err == hipSuccess ? FA_OK : FA_ERR_HIP;
}

// Grid checks of the decode-shaped path (after check_fused and the degenerate sizes), and the bytes of
// partial results it stores (-1 if the count overflows).
fa_status_t decode_grid(int B, int Hq, int Hkv, int Sq, int d_v, int n_parts, int64_t* need) {
  const int64_t n_cb = (static_cast<int64_t>(Hq / Hkv) * Sq + 31) / 32;
  if (static_cast<int64_t>(B) * Hkv * n_cb * n_parts > INT_MAX || static_cast<int64_t>(B) * Hq * Sq > INT_MAX)
    return FA_ERR_BAD_SHAPE;
  *need = split_workspace_bytes(B, Hq, Sq, d_v, n_parts);
  return FA_OK;
}

hipError_t decode_launch(const void* Q, const void* K, const void* V, void* O, float* LSE, int B, int Hq, int Hkv,
                         int Sq, int Sk, int d_qk, int d_v, float cs, int causal, int n_parts, void* ws,
                         hipStream_t stream) {
  fa::DecodeParams p{};
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
  p.causal = causal != 0;
  p.cs = cs;
  p.rows = p.group * Sq;
  p.n_parts = n_parts;
  const int64_t rows = static_cast<int64_t>(B) * Hq * Sq;
  p.o_part = static_cast<float*>(ws);
  p.lse_part = p.o_part + rows * n_parts * d_v;
  return fa::launch_decode(p, d_qk, d_v, stream);
}

// ---- per-device address of the static scratch (declared at the top of the file) -------------------

constexpr int kMaxDevices = 64;
std::atomic<void*> g_scratch[kMaxDevices];
std::mutex g_scratch_mu;

// Device address of `scratch` on the device `stream` belongs to (the current device for the null
// stream). The first call on a device looks it up; later calls read the cached address.
hipError_t scratch_for_stream(hipStream_t stream, void** out) {
  int cur = 0;
  hipError_t e = hipGetDevice(&cur);
  if (e != hipSuccess) return e;
  int dev = cur;
  if (stream != nullptr) {
    e = hipStreamGetDevice(stream, &dev);
    if (e != hipSuccess) return e;
  }
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  void* ptr = g_scratch[dev].load(std::memory_order_acquire);
  if (ptr != nullptr) {
    *out = ptr;
    return hipSuccess;
  }
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  ptr = g_scratch[dev].load(std::memory_order_relaxed);
  if (ptr == nullptr) {
    if (dev != cur && (e = hipSetDevice(dev)) != hipSuccess) return e;
    e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (dev != cur) {
      const hipError_t e2 = hipSetDevice(cur);
      if (e == hipSuccess) e = e2;
    }
    if (e != hipSuccess || ptr == nullptr) return e != hipSuccess ? e : hipErrorInvalidSymbol;
    g_scratch[dev].store(ptr, std::memory_order_release);
  }
  *out = ptr;
  return hipSuccess;
}

// ---- layer-by-layer operators ------------------------------------------------------------------

int64_t lbl_ld(int Sk) { return (static_cast<int64_t>(Sk) + fa::kLblKeys - 1) / fa::kLblKeys * fa::kLblKeys; }

// Shared checks of the layer-by-layer entry points, in the order documented in fa.h. d_qk / d_v are
// checked only where the operator uses them (0 = unused).
fa_status_t lbl_check_shape(int B, int Hq, int Hkv, int Sq, int Sk, int d_qk, int d_v) {
  if (B < 0 || Hq < 0 || Hkv < 0 || Sq < 0 || Sk < 0) return FA_ERR_BAD_SHAPE;
  if (Hq > 0 && (Hkv <= 0 || Hq % Hkv != 0)) return FA_ERR_BAD_SHAPE;
  if (Sk > fa::kLblMaxSk) return FA_ERR_BAD_SHAPE;
  const int64_t dmax = d_qk > d_v ? d_qk : d_v;
  if (static_cast<int64_t>(Sq) * dmax > INT_MAX || static_cast<int64_t>(Sk) * dmax > INT_MAX) return FA_ERR_BAD_SHAPE;
  const int64_t n_qb = (static_cast<int64_t>(Sq) + fa::kLblRows - 1) / fa::kLblRows;
  if (static_cast<int64_t>(B) * Hq * n_qb > INT_MAX) return FA_ERR_BAD_SHAPE;
  if (static_cast<int64_t>(B) * Hq * Sq > 4 * static_cast<int64_t>(INT_MAX)) return FA_ERR_BAD_SHAPE;
  if (static_cast<int64_t>(B) * Hkv > INT_MAX) return FA_ERR_BAD_SHAPE;
  if (d_qk != 0 && !fa::lbl_scores_supported(d_qk)) return FA_ERR_UNSUPPORTED;
  if (d_v != 0 && !fa::lbl_pv_supported(d_v)) return FA_ERR_UNSUPPORTED;
  return FA_OK;
}

// The whole problem as one chunk; spill buffers S and P.
fa::LblParams lbl_params(int B, int Hq, int Hkv, int Sq, int Sk, float scale, int causal) {
  fa::LblParams p{};
  p.batch = B;
  p.hq = Hq;
  p.hkv = Hkv;
  p.sq = Sq;
  p.sk = Sk;
  p.group = Hkv > 0 ? Hq / Hkv : 1;
  p.causal = causal != 0;
  p.ld = static_cast<int>(lbl_ld(Sk));
  p.scale = scale;
  p.bh0 = 0;
  p.nbh = B * Hq;
  p.qb0 = 0;
  p.nqb = (Sq + fa::kLblRows - 1) / fa::kLblRows;
  p.xgroup = p.group;
  p.rows = static_cast<int64_t>(B) * Hq * Sq;
  return p;
}

}  // namespace

extern "C" {

fa_status_t fa_fwd_ex(const void* Q, const void* K, const void* V, void* O, float* LSE, int B, int Hq, int Hkv,
                      int Sq, int Sk, int d_qk, int d_v, float scale, int causal, hipStream_t stream) {
  return forward(Q, K, V, O, LSE, B, Hq, Hkv, Sq, Sk, d_qk, d_v, scale, causal, stream);
}

fa_status_t fa_fwd(const void* Q, const void* K, const void* V, void* O, int B, int Hq, int Hkv, int Sq, int Sk,
                   int d, float scale, int causal, hipStream_t stream) {
  return forward(Q, K, V, O, nullptr, B, Hq, Hkv, Sq, Sk, d, d, scale, causal, stream);
}

fa_status_t fa_fwd_split(const void* Q, const void* K, const void* V, void* O, float* LSE, int B, int Hq, int Hkv,
                         int Sq, int Sk, int d_qk, int d_v, float scale, int causal, int n_split, void* workspace,
                         size_t workspace_bytes, hipStream_t stream) {
  if (n_split < 1) return FA_ERR_BAD_SHAPE;
  return forward(Q, K, V, O, LSE, B, Hq, Hkv, Sq, Sk, d_qk, d_v, scale, causal, stream, n_split, workspace,
                 workspace_bytes);
}

fa_status_t fa_fwd_decode(const void* Q, const void* K, const void* V, void* O, float* LSE, int B, int Hq, int Hkv,
                          int Sq, int Sk, int d_qk, int d_v, float scale, int causal, int n_parts, void* workspace,
                          size_t workspace_bytes, hipStream_t stream) {
  if (n_parts < 1) return FA_ERR_BAD_SHAPE;
  float cs = 0.f;
  fa_status_t st = check_fused(Q, K, V, O, LSE, B, Hq, Hkv, Sq, Sk, d_qk, d_v, scale, causal, &cs);
  if (st != FA_OK) return st;
  if (static_cast<int64_t>(B) * Hq * Sq == 0) return FA_OK;
  int64_t need = 0;
  st = decode_grid(B, Hq, Hkv, Sq, d_v, n_parts, &need);
  if (st != FA_OK) return st;
  if (need < 0 || workspace == nullptr || static_cast<uint64_t>(need) > workspace_bytes) return FA_ERR_WORKSPACE;
  if (!aligned(workspace, 16)) return FA_ERR_UNSUPPORTED;
  return decode_launch(Q, K, V, O, LSE, B, Hq, Hkv, Sq, Sk, d_qk, d_v, cs, causal, n_parts, workspace, stream) ==
                 hipSuccess
             ? FA_OK
             : FA_ERR_HIP;
}

fa_status_t fa_fwd_decode_noalloc(const void* Q, const void* K, const void* V, void* O, float* LSE, int B, int Hq,
                                  int Hkv, int Sq, int Sk, int d_qk, int d_v, float scale, int causal, int n_parts,
                                  hipStream_t stream) {
  if (n_parts < 1) return FA_ERR_BAD_SHAPE;
  float cs = 0.f;
  fa_status_t st = check_fused(Q, K, V, O, LSE, B, Hq, Hkv, Sq, Sk, d_qk, d_v, scale, causal, &cs);
  if (st != FA_OK) return st;
  if (static_cast<int64_t>(B) * Hq * Sq == 0) return FA_OK;
  int64_t need = 0;
  st = decode_grid(B, Hq, Hkv, Sq, d_v, n_parts, &need);
  if (st != FA_OK) return st;
  if (need < 0 || need > static_cast<int64_t>(FA_NOALLOC_SCRATCH_BYTES)) return FA_ERR_WORKSPACE;
  void* ws = nullptr;
  if (scratch_for_stream(stream, &ws) != hipSuccess) return FA_ERR_HIP;
  return decode_launch(Q, K, V, O, LSE, B, Hq, Hkv, Sq, Sk, d_qk, d_v, cs, causal, n_parts, ws, stream) ==
                 hipSuccess
             ? FA_OK
             : FA_ERR_HIP;
}

int fa_fwd_decode_parts(int n_cu, int B, int Hq, int Hkv, int Sq, int Sk) {
  if (n_cu <= 0 || B <= 0 || Hq <= 0 || Hkv <= 0 || Hq % Hkv != 0 || Sq <= 0 || Sk < 0) return 0;
  // One workgroup per CU in total (a workgroup holds two K+V tiles in LDS, so one fits a CU), but
  // no part shorter than 4 key tiles.
  const int64_t n_cb = (static_cast<int64_t>(Hq / Hkv) * Sq + 31) / 32;
  const int64_t items = static_cast<int64_t>(B) * Hkv * n_cb;
  const int64_t tiles = (static_cast<int64_t>(Sk) + fa::decode_tile_keys() - 1) / fa::decode_tile_keys();
  int64_t parts = (n_cu + items - 1) / items;
  const int64_t max_parts = (tiles + 3) / 4;
  if (parts > max_parts) parts = max_parts;
  return parts < 1 ? 1 : static_cast<int>(parts);
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

int fa_lbl_ld(int Sk) { return Sk < 0 || Sk > fa::kLblMaxSk ? -1 : static_cast<int>(lbl_ld(Sk)); }

size_t fa_lbl_workspace_bytes(int B, int Hq, int Sq, int Sk) {
  if (B <= 0 || Hq <= 0 || Sq <= 0 || Sk <= 0) return 0;
  if (Sk > fa::kLblMaxSk) return SIZE_MAX;
  const int64_t bh = static_cast<int64_t>(B) * Hq;
  const int64_t per_row = lbl_ld(Sk) * 2;  // < 2^24
  if (bh > INT64_MAX / Sq) return SIZE_MAX;
  const int64_t rows = bh * Sq;
  if (rows > INT64_MAX / per_row) return SIZE_MAX;
  return static_cast<size_t>(rows * per_row);
}

fa_status_t fa_lbl_scores(const void* Q, const void* K, void* S, int B, int Hq, int Hkv, int Sq, int Sk, int d_qk,
                          float scale, int causal, hipStream_t stream) {
  fa_status_t st = lbl_check_shape(B, Hq, Hkv, Sq, Sk, d_qk, 0);
  if (st != FA_OK) return st;
  const bool q_rows = static_cast<int64_t>(B) * Hq * Sq > 0;
  const bool kv_rows = static_cast<int64_t>(B) * Hkv * Sk > 0;
  if ((q_rows && Q == nullptr) || (kv_rows && K == nullptr) || (q_rows && Sk > 0 && S == nullptr))
    return FA_ERR_NULL_POINTER;
  if (!isfinite(scale)) return FA_ERR_BAD_SCALE;
  if (!aligned(Q, 16) || !aligned(K, 16) || !aligned(S, 16)) return FA_ERR_UNSUPPORTED;
  if (!q_rows || Sk == 0) return FA_OK;  // no score to write
  fa::LblParams p = lbl_params(B, Hq, Hkv, Sq, Sk, scale, causal);
  p.q = static_cast<const uint16_t*>(Q);
  p.k = static_cast<const uint16_t*>(K);
  p.s = static_cast<uint16_t*>(S);
  return fa::launch_lbl_scores(p, d_qk, stream) == hipSuccess ? FA_OK : FA_ERR_HIP;
}

fa_status_t fa_lbl_softmax(const void* S, void* P, float* LSE, int B, int Hq, int Sq, int Sk, int causal,
                           hipStream_t stream) {
  fa_status_t st = lbl_check_shape(B, Hq, Hq > 0 ? 1 : 0, Sq, Sk, 0, 0);
  if (st != FA_OK) return st;
  const bool rows = static_cast<int64_t>(B) * Hq * Sq > 0;
  if (rows && Sk > 0 && (S == nullptr || P == nullptr)) return FA_ERR_NULL_POINTER;
  if (!aligned(S, 16) || !aligned(P, 16) || !aligned(LSE, 4)) return FA_ERR_UNSUPPORTED;
  if (!rows) return FA_OK;
  fa::LblParams p = lbl_params(B, Hq, 1, Sq, Sk, 1.f, causal);
  p.s = const_cast<uint16_t*>(static_cast<const uint16_t*>(S));
  p.p = static_cast<uint16_t*>(P);
  p.lse = LSE;
  return fa::launch_lbl_softmax(p, stream) == hipSuccess ? FA_OK : FA_ERR_HIP;
}

fa_status_t fa_lbl_pv(const void* P, const void* V, void* O, int B, int Hq, int Hkv, int Sq, int Sk, int d_v,
                      int causal, hipStream_t stream) {
  fa_status_t st = lbl_check_shape(B, Hq, Hkv, Sq, Sk, 0, d_v);
  if (st != FA_OK) return st;
  const bool q_rows = static_cast<int64_t>(B) * Hq * Sq > 0;
  const bool kv_rows = static_cast<int64_t>(B) * Hkv * Sk > 0;
  if ((q_rows && O == nullptr) || (kv_rows && V == nullptr) || (q_rows && Sk > 0 && P == nullptr))
    return FA_ERR_NULL_POINTER;
  if (!aligned(P, 16) || !aligned(V, 16) || !aligned(O, 16)) return FA_ERR_UNSUPPORTED;
  if (!q_rows) return FA_OK;
  fa::LblParams p = lbl_params(B, Hq, Hkv, Sq, Sk, 1.f, causal);
  p.p = const_cast<uint16_t*>(static_cast<const uint16_t*>(P));
  p.v = static_cast<const uint16_t*>(V);
  p.o = static_cast<uint16_t*>(O);
  return fa::launch_lbl_pv(p, d_v, stream) == hipSuccess ? FA_OK : FA_ERR_HIP;
}

fa_status_t fa_fwd_unfused(const void* Q, const void* K, const void* V, void* O, float* LSE, int B, int Hq, int Hkv,
                           int Sq, int Sk, int d_qk, int d_v, float scale, int causal, void* workspace,
                           size_t workspace_bytes, hipStream_t stream) {
  fa_status_t st = lbl_check_shape(B, Hq, Hkv, Sq, Sk, d_qk, d_v);
  if (st != FA_OK) return st;
  const bool q_rows = static_cast<int64_t>(B) * Hq * Sq > 0;
  const bool kv_rows = static_cast<int64_t>(B) * Hkv * Sk > 0;
  if ((q_rows && (Q == nullptr || O == nullptr)) || (kv_rows && (K == nullptr || V == nullptr)))
    return FA_ERR_NULL_POINTER;
  if (!isfinite(scale)) return FA_ERR_BAD_SCALE;
  if (!aligned(Q, 16) || !aligned(K, 16) || !aligned(V, 16) || !aligned(O, 16) || !aligned(LSE, 4))
    return FA_ERR_UNSUPPORTED;
  if (!q_rows) return FA_OK;
  // Rows of spill buffer the workspace holds; one block of query rows (or all of Sq if shorter) is
  // the least a chunk needs.
  const int64_t row_bytes = lbl_ld(Sk) * 2;
  const int64_t min_rows = Sq < fa::kLblRows ? Sq : fa::kLblRows;
  const int64_t cap = row_bytes == 0 ? INT64_MAX : static_cast<int64_t>(workspace_bytes / row_bytes);
  if (row_bytes > 0 && (workspace == nullptr || cap < min_rows)) return FA_ERR_WORKSPACE;
  if (!aligned(workspace, 16)) return FA_ERR_UNSUPPORTED;

  fa::LblParams p = lbl_params(B, Hq, Hkv, Sq, Sk, scale, causal);
  p.q = static_cast<const uint16_t*>(Q);
  p.k = static_cast<const uint16_t*>(K);
  p.v = static_cast<const uint16_t*>(V);
  p.o = static_cast<uint16_t*>(O);
  p.lse = LSE;
  p.s = p.p = static_cast<uint16_t*>(workspace);  // probabilities overwrite the scores in place
  const int n_bh = B * Hq, n_qb = p.nqb;
  const hipStream_t s = stream;
  auto run = [&](int bh0, int nbh, int qb0, int nqb) {
    p.bh0 = bh0;
    p.nbh = nbh;
    p.qb0 = qb0;
    p.nqb = nqb;
    p.xgroup = (bh0 % p.group == 0 && nbh % p.group == 0) ? p.group : 1;
    const int64_t last = static_cast<int64_t>(qb0 + nqb) * fa::kLblRows;
    p.rows = static_cast<int64_t>(nbh - 1) * Sq + (last < Sq ? last : Sq) - static_cast<int64_t>(qb0) * fa::kLblRows;
    if (fa::launch_lbl_scores(p, d_qk, s) != hipSuccess) return false;
    if (fa::launch_lbl_softmax(p, s) != hipSuccess) return false;
    return fa::launch_lbl_pv(p, d_v, s) == hipSuccess;
  };
  if (cap >= static_cast<int64_t>(Sq)) {
    // Whole heads per chunk, a multiple of the group size when more than one group fits.
    int64_t heads = cap / Sq;
    if (heads > n_bh) heads = n_bh;
    if (heads >= p.group) heads -= heads % p.group;
    for (int64_t bh0 = 0; bh0 < n_bh; bh0 += heads) {  // 64-bit: bh0 + heads may pass INT_MAX
      const int nbh = static_cast<int>(n_bh - bh0 < heads ? n_bh - bh0 : heads);
      if (!run(static_cast<int>(bh0), nbh, 0, n_qb)) return FA_ERR_HIP;
    }
  } else {
    // Part of one head per chunk.
    const int blocks = static_cast<int>(cap / fa::kLblRows);
    for (int bh = 0; bh < n_bh; ++bh)
      for (int qb0 = 0; qb0 < n_qb; qb0 += blocks)
        if (!run(bh, 1, qb0, n_qb - qb0 < blocks ? n_qb - qb0 : blocks)) return FA_ERR_HIP;
  }
  return FA_OK;
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

int fa_fwd_rows(int B, int Hq, int Sq, int d_qk, int d_v, int causal) {
  return fa::instance_rows(B, Hq, Sq, d_qk, d_v, causal != 0);
}

}  // extern "C"
