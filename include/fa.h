/*
 * fa.h -- C ABI of the fused attention forward for AMD Instinct MI355X (gfx950).
 *
 * Operation (the paper's scaled dot-product attention, Eq. (1), Sec. 2.1, replicated over heads):
 *
 *     O[b,h] = softmax(scale * Q[b,h] * K[b,g]^T) * V[b,g],   g = h / (Hq / Hkv)
 *
 * computed in one kernel launch: the score tile S = Q K^T never leaves the chip; an online softmax
 * keeps a running row max and row sum and rescales the partial P V accumulation (Alg. 1, Sec. 2.1).
 * The query heads h of one group share key/value head g (grouped-query attention, Sec. 4.4 and
 * Sec. 6.5). With causal masking, key j is visible to query i iff j <= i + (Sk - Sq) (bottom-right
 * alignment; the usual j <= i when Sq == Sk).
 *
 * Element types: Q, K, V and O are IEEE bfloat16 bit patterns (torch.bfloat16). LSE is float32.
 * Arithmetic: bf16 x bf16 products with fp32 accumulation for both contractions; softmax statistics
 * and the output accumulator in fp32; P is rounded to bf16 (round-to-nearest-even) only as the
 * operand of the P V product; O is rounded to bf16 (RNE) once, at the end.
 *
 * Layout: every tensor is a contiguous row-major BHSD array in device memory, no strides:
 *     Q   [B][Hq ][Sq][d_qk]      K [B][Hkv][Sk][d_qk]      V [B][Hkv][Sk][d_v]
 *     O   [B][Hq ][Sq][d_v ]      LSE (optional) float32 [B][Hq][Sq]
 * LSE[b,h,i] = ln( sum over visible j of exp(scale * q_i . k_j) ), natural log; -inf for a row with
 * no visible key (that row's O is 0).
 *
 * Ownership: the caller owns every buffer. The library allocates nothing, frees nothing, keeps no
 * state beyond its compiled kernels, and is reentrant and thread-safe. Q, K, V are only read; O and
 * LSE are only written, every element exactly once per call.
 *
 * Asynchrony: the work is enqueued on `stream` (a hipStream_t passed as void*; NULL is the null
 * stream of the current device); FA_OK means "enqueued". The library never synchronises. Faults
 * during execution surface at the caller's next synchronisation.
 *
 * Errors: every argument check runs on the host before any HIP call. On any error return nothing is
 * launched and O / LSE are untouched, so the checks are usable on a machine without a GPU. Checks run
 * in this order and the first failing one is reported: sizes (FA_ERR_BAD_SHAPE), head dimensions
 * (FA_ERR_UNSUPPORTED), pointers (FA_ERR_NULL_POINTER), scale (FA_ERR_BAD_SCALE), alignment
 * (FA_ERR_UNSUPPORTED), index ranges (FA_ERR_BAD_SHAPE).
 *
 * Degenerate sizes: B == 0, Hq == 0 or Sq == 0 is a no-op returning FA_OK (no HIP call). Sk == 0
 * is valid: every row gets O = 0 and LSE = -inf.
 *
 * Supported head dimensions: (d_qk, d_v) in {(64, 64), (128, 128), (192, 128)}; others return
 * FA_ERR_UNSUPPORTED.
 */
#ifndef FA_MI355X_FA_H
#define FA_MI355X_FA_H

#include <stddef.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  FA_OK = 0,
  FA_ERR_NULL_POINTER = 1, /* Q or O is NULL with B*Hq*Sq > 0, or K or V is NULL with B*Hkv*Sk > 0 */
                           /* (LSE may always be NULL)                                            */
  FA_ERR_BAD_SHAPE = 2,    /* a size < 0; Hkv <= 0 or Hq % Hkv != 0 with Hq > 0; Sq*d or Sk*d of  */
                           /* one head >= 2^31 elements; more than 2^31-1 workgroups              */
  FA_ERR_UNSUPPORTED = 3,  /* (d_qk, d_v) not compiled in; Q/K/V/O not 16-byte aligned, or LSE   */
                           /* not 4-byte aligned                                                  */
  FA_ERR_BAD_SCALE = 4,    /* scale is NaN or +-inf, or |scale| * log2(e) overflows float32       */
  FA_ERR_HIP = 5,          /* the HIP runtime reported an error when enqueuing the kernel         */
  FA_ERR_WORKSPACE = 6     /* split mode: workspace NULL or smaller than                          */
                           /* fa_fwd_split_workspace_bytes(B, Hq, Sq, d_v, n_split)               */
} fa_status_t;

/*
 * fa_fwd -- attention forward with one head dimension d = d_qk = d_v and no LSE output.
 * Same contract as fa_fwd_ex(Q, K, V, O, NULL, B, Hq, Hkv, Sq, Sk, d, d, scale, causal, stream).
 */
fa_status_t fa_fwd(const void* Q, const void* K, const void* V, void* O, int B, int Hq, int Hkv,
                   int Sq, int Sk, int d, float scale, int causal, void* stream);

/*
 * fa_fwd_ex -- general entry point.
 *   Q, K, V   device pointers to bf16 inputs (layout above), 16-byte aligned
 *   O         device pointer to the bf16 output, 16-byte aligned
 *   LSE       device pointer to the float32 log-sum-exp output, 4-byte aligned, or NULL to skip it
 *   B, Hq, Hkv, Sq, Sk   batch, query heads, key/value heads, query length, key length (>= 0)
 *   d_qk, d_v head dimension of Q/K and of V/O
 *   scale     multiplier of the scores (the paper uses 1/sqrt(d_k)); any finite value, including
 *             0 (uniform weights over the visible keys) and negative values
 *   causal    nonzero for bottom-right causal masking
 *   stream    hipStream_t to enqueue on
 */
fa_status_t fa_fwd_ex(const void* Q, const void* K, const void* V, void* O, float* LSE, int B,
                      int Hq, int Hkv, int Sq, int Sk, int d_qk, int d_v, float scale, int causal,
                      void* stream);

/*
 * fa_fwd_split -- the same operation with every query block's key range cut into n_split parts that
 * run as separate workgroups, for shapes with too few query blocks to fill the GPU (short or few
 * query rows against long keys). This is the paper's tile-to-tile level (Alg. 2, Sec. 2.1): each
 * part runs the per-tile online softmax (Alg. 1) over its contiguous run of 64-key tiles and yields a
 * partial result; a second kernel merges the parts of every row with the log-sum-exp combination
 * (u = max over parts of u_c; each part's accumulator and row sum rescaled by exp(u_c - u) before
 * they are added), then normalises. Results agree with fa_fwd_ex within floating-point rounding.
 *
 *   Q .. stream  as in fa_fwd_ex
 *   n_split      parts per query block (>= 1). Each query block's visible key tiles are divided into
 *                n_split runs of ceil(tiles / n_split) tiles; parts left without a tile contribute
 *                nothing.
 *   workspace    device buffer owned by the caller, 16-byte aligned, at least
 *                fa_fwd_split_workspace_bytes(B, Hq, Sq, d_v, n_split) bytes; overwritten by the call
 *                (fp32 partial outputs [n_split][B][Hq][Sq][d_v], then partial LSE
 *                [n_split][B][Hq][Sq]); the caller must not touch it until the call's work on
 *                `stream` has completed. NULL is allowed only when no byte is needed.
 *   workspace_bytes  its size in bytes
 *
 * Enqueues two kernels on `stream`. Errors: n_split < 1 first (FA_ERR_BAD_SHAPE), then the checks of
 * fa_fwd_ex in their order (a degenerate size still returns FA_OK without touching the workspace),
 * then more than 2^31-1 workgroups in total (FA_ERR_BAD_SHAPE), workspace NULL or too small
 * (FA_ERR_WORKSPACE), workspace not 16-byte aligned (FA_ERR_UNSUPPORTED).
 */
fa_status_t fa_fwd_split(const void* Q, const void* K, const void* V, void* O, float* LSE, int B,
                         int Hq, int Hkv, int Sq, int Sk, int d_qk, int d_v, float scale, int causal,
                         int n_split, void* workspace, size_t workspace_bytes, void* stream);

/* Workspace bytes fa_fwd_split needs: n_split * B * Hq * Sq * (d_v + 1) * 4; 0 when B, Hq, Sq, d_v
 * or n_split is <= 0 (nothing to store); SIZE_MAX if the count overflows. */
size_t fa_fwd_split_workspace_bytes(int B, int Hq, int Sq, int d_v, int n_split);

/* Suggested n_split for fa_fwd_split on a device with n_cu compute units: about two workgroups per
 * CU over all parts, no part shorter than 8 key tiles (512 keys), at least 1 (1 means the single
 * pass fa_fwd_ex is the better call). Host arithmetic only, no HIP call. Returns 0 for unsupported
 * head dimensions or n_cu, B, Hq, Sq <= 0 or Sk < 0. */
int fa_fwd_split_parts(int n_cu, int B, int Hq, int Sq, int Sk, int d_qk, int d_v, int causal);

/* Static, human-readable name of a status code ("FA_OK", ...); "unknown status" otherwise. */
const char* fa_status_str(fa_status_t s);

/* Number of query rows one workgroup processes for the given head dimensions (0 if unsupported). */
int fa_block_rows(int d_qk, int d_v, int causal);

#ifdef __cplusplus
}
#endif

#endif /* FA_MI355X_FA_H */
