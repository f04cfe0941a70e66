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

fa_status_t forward(const void* Q, const void* K, const void* V, void* O, float* LSE, int B, int Hq, int Hkv,
                    int Sq, int Sk, int d_qk, int d_v, float scale, int causal, void* stream) {
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
  const hipError_t err = fa::launch_forward(p, d_qk, d_v, causal != 0, static_cast<hipStream_t>(stream));
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

const char* fa_status_str(fa_status_t s) {
  switch (s) {
    case FA_OK: return "FA_OK";
    case FA_ERR_NULL_POINTER: return "FA_ERR_NULL_POINTER";
    case FA_ERR_BAD_SHAPE: return "FA_ERR_BAD_SHAPE";
    case FA_ERR_UNSUPPORTED: return "FA_ERR_UNSUPPORTED";
    case FA_ERR_BAD_SCALE: return "FA_ERR_BAD_SCALE";
    case FA_ERR_HIP: return "FA_ERR_HIP";
  }
  return "unknown status";
}

int fa_block_rows(int d_qk, int d_v, int causal) { return fa::block_rows(d_qk, d_v, causal != 0); }

}  // extern "C"
