/*
 * fa.h -- C ABI of the attention forward for AMD Instinct MI355X (gfx950): the fused kernel, its
 * split mode, and the unfused layer-by-layer operators it is measured against.
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
 * Ownership: the caller owns every buffer. The library allocates nothing, frees nothing, and is
 * reentrant and thread-safe; its only state is the static scratch array of fa_fwd_decode_noalloc
 * (below) and that array's per-device address. Q, K, V are only read; O and
 * LSE are only written, every element exactly once per call.
 *
 * Asynchrony: the work is enqueued on `stream` (NULL is the null stream of the current device);
 * FA_OK means "enqueued". The library never synchronises. Faults
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

/* HIP's stream handle, the same declaration as in hip/hip_runtime_api.h, so that this header needs
 * no HIP include (C callers may include either header first). */
typedef struct ihipStream_t* hipStream_t;

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
                           /* fa_fwd_split_workspace_bytes(B, Hq, Sq, d_v, n_split); for          */
                           /* fa_fwd_decode_noalloc: that size exceeds FA_NOALLOC_SCRATCH_BYTES   */
} fa_status_t;

/*
 * fa_fwd -- attention forward with one head dimension d = d_qk = d_v and no LSE output.
 * Same contract as fa_fwd_ex(Q, K, V, O, NULL, B, Hq, Hkv, Sq, Sk, d, d, scale, causal, stream).
 */
fa_status_t fa_fwd(const void* Q, const void* K, const void* V, void* O, int B, int Hq, int Hkv,
                   int Sq, int Sk, int d, float scale, int causal, hipStream_t stream);

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
 *   stream    the HIP stream to enqueue on
 */
fa_status_t fa_fwd_ex(const void* Q, const void* K, const void* V, void* O, float* LSE, int B,
                      int Hq, int Hkv, int Sq, int Sk, int d_qk, int d_v, float scale, int causal,
                      hipStream_t stream);

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
 * then more than 2^31-1 workgroups in total or more than 2^31-1 rows B*Hq*Sq (FA_ERR_BAD_SHAPE),
 * workspace NULL or too small (FA_ERR_WORKSPACE), workspace not 16-byte aligned (FA_ERR_UNSUPPORTED).
 */
fa_status_t fa_fwd_split(const void* Q, const void* K, const void* V, void* O, float* LSE, int B,
                         int Hq, int Hkv, int Sq, int Sk, int d_qk, int d_v, float scale, int causal,
                         int n_split, void* workspace, size_t workspace_bytes, hipStream_t stream);

/* Workspace bytes fa_fwd_split needs: n_split * B * Hq * Sq * (d_v + 1) * 4; 0 when B, Hq, Sq, d_v
 * or n_split is <= 0 (nothing to store); SIZE_MAX if the count overflows. */
size_t fa_fwd_split_workspace_bytes(int B, int Hq, int Sq, int d_v, int n_split);

/*
 * fa_fwd_decode -- the same operation for decode-shaped problems, where each key/value head has few
 * query rows (one to a few new tokens per query head; best when (Hq / Hkv) * Sq <= 32). The Hq / Hkv
 * query heads that share a key/value head and their Sq rows are computed together as the columns of
 * 32-column matrix-core blocks, so K and V are read once per key/value head and block of 32 rows.
 * The key range of every (batch, key/value head, block) is cut into n_parts contiguous runs of
 * 128-key tiles that run as separate
 * workgroups (the tile-to-tile level, Alg. 2, Sec. 2.1), each running the per-tile online softmax
 * (Alg. 1); a second kernel merges the parts with the log-sum-exp combination, as fa_fwd_split does.
 * Results agree with fa_fwd_ex within floating-point rounding.
 *
 *   Q .. stream  as in fa_fwd_ex
 *   n_parts      key-range parts per (batch, key/value head, block), >= 1; parts left without a tile
 *                contribute nothing. fa_fwd_decode_parts suggests a count.
 *   workspace    device buffer owned by the caller, 16-byte aligned, at least
 *                fa_fwd_split_workspace_bytes(B, Hq, Sq, d_v, n_parts) bytes, with the layout of
 *                fa_fwd_split's workspace; overwritten by the call and not to be touched until the
 *                call's work on `stream` has completed. NULL only when no byte is needed.
 *   workspace_bytes  its size in bytes
 *
 * Enqueues two kernels on `stream`. Errors: n_parts < 1 (FA_ERR_BAD_SHAPE); then sizes
 * (FA_ERR_BAD_SHAPE), head dimensions (FA_ERR_UNSUPPORTED), pointers
 * (FA_ERR_NULL_POINTER), scale (FA_ERR_BAD_SCALE), alignment (FA_ERR_UNSUPPORTED), index ranges
 * (FA_ERR_BAD_SHAPE); B*Hq*Sq == 0 returns FA_OK without touching the workspace; then more than
 * 2^31-1 workgroups or 2^31-1 rows B*Hq*Sq (FA_ERR_BAD_SHAPE), workspace NULL or too small
 * (FA_ERR_WORKSPACE), workspace not 16-byte aligned (FA_ERR_UNSUPPORTED).
 */
fa_status_t fa_fwd_decode(const void* Q, const void* K, const void* V, void* O, float* LSE, int B,
                          int Hq, int Hkv, int Sq, int Sk, int d_qk, int d_v, float scale, int causal,
                          int n_parts, void* workspace, size_t workspace_bytes, hipStream_t stream);

/* Bytes of the static scratch array behind fa_fwd_decode_noalloc (32 MiB per device). */
#define FA_NOALLOC_SCRATCH_BYTES (32u << 20)

/*
 * fa_fwd_decode_noalloc -- fa_fwd_decode for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc): the same kernels and
 * results, bit for bit, as fa_fwd_decode with the same n_parts, but the partial results live in a
 * static device array of FA_NOALLOC_SCRATCH_BYTES that the library holds on every device it runs on
 * until the process ends, instead of a caller workspace. The call allocates and frees nothing.
 *
 *   Q .. causal, n_parts   as in fa_fwd_decode
 *   stream                 the HIP stream to enqueue on; the scratch of the stream's device is used
 *                          (the current device's for the NULL stream)
 *
 * The first call on a device looks up that device's scratch address (hipGetSymbolAddress), once.
 * Every call on one device shares its scratch, and every element a call reads there it has written
 * itself first (nothing needs to start at zero). Calls that overlap in time on one device -- on two
 * streams, or from two threads without ordering -- race on the scratch and give undefined results;
 * calls ordered on one stream do not.
 *
 * Errors: n_parts < 1 (FA_ERR_BAD_SHAPE); then the checks of fa_fwd_decode in their order up to the
 * grid size (B*Hq*Sq == 0 returns FA_OK with no HIP call); then partial results of
 * fa_fwd_split_workspace_bytes(B, Hq, Sq, d_v, n_parts) > FA_NOALLOC_SCRATCH_BYTES bytes
 * (FA_ERR_WORKSPACE: fewer parts, or fa_fwd_decode with a workspace, is the remedy); a failed lookup
 * of the scratch address or a failed launch (FA_ERR_HIP).
 */
fa_status_t fa_fwd_decode_noalloc(const void* Q, const void* K, const void* V, void* O, float* LSE, int B,
                                  int Hq, int Hkv, int Sq, int Sk, int d_qk, int d_v, float scale,
                                  int causal, int n_parts, hipStream_t stream);

/* Suggested n_parts for fa_fwd_decode on a device with n_cu compute units: about one workgroup per
 * CU in total, no part shorter than 4 key tiles (512 keys), at least 1. Host arithmetic only.
 * Returns 0 if n_cu, B, Hq, Hkv or Sq <= 0, Hq % Hkv != 0 or Sk < 0. */
int fa_fwd_decode_parts(int n_cu, int B, int Hq, int Hkv, int Sq, int Sk);

/* Suggested n_split for fa_fwd_split on a device with n_cu compute units: about two workgroups per
 * CU over all parts, no part shorter than 8 key tiles (512 keys), at least 1 (1 means the single
 * pass fa_fwd_ex is the better call). Host arithmetic only, no HIP call. Returns 0 for unsupported
 * head dimensions or n_cu, B, Hq, Sq <= 0 or Sk < 0. */
int fa_fwd_split_parts(int n_cu, int B, int Hq, int Sq, int Sk, int d_qk, int d_v, int causal);

/*
 * Layer-by-layer (unfused) attention -- the paper's diagnostic baseline mapping (Sec. "Diagnostic
 * Baseline: Unfused Layer-by-Layer Attention"): the same operation as three operators dispatched
 * one after another, each reading its input from device memory and writing its result back, with
 * the intermediates in bfloat16 (Table 3 lists the score matrix QK^T and the probability matrix
 * among what this mapping spills):
 *
 *   fa_lbl_scores:   S[b,h,i,j] = bf16(scale * q_i . k_j)                (fp32 accumulation, RNE)
 *   fa_lbl_softmax:  LSE[b,h,i] = ln sum over visible j of exp(S[b,h,i,j]);
 *                    P[b,h,i,j] = bf16(exp(S[b,h,i,j] - LSE[b,h,i])) for visible j, 0 for masked j
 *   fa_lbl_pv:       O[b,h,i,:] = bf16(sum over j of P[b,h,i,j] * V[b,g,j,:])  (fp32 accumulation)
 *
 * It exists to measure what fusion saves; fa_fwd_ex is the operation's fast path. Results differ
 * from fa_fwd_ex by the roundings of S and P: per output row at most
 * max|V| * ((1 + u)^2 * exp(2 u M) - 1) with u = 2^-8 and M the row's largest visible |score|, plus
 * fp32 accumulation error.
 *
 * Spill buffers S and P: bf16 [B][Hq][Sq][ld] with row stride ld = fa_lbl_ld(Sk) (Sk rounded up to
 * 64), 16-byte aligned, owned by the caller. Row extents: query rows are taken in blocks of 128
 * (rows 128*c .. 128*c+127 of a head); let n be the number of keys visible to the last row of the
 * block (Sk without causal masking); the block's extent is E = 64 * ceil(n / 64) <= ld.
 *   - fa_lbl_scores writes S[i][j] for j < E (unmasked values, also past the diagonal) and nothing
 *     else of S;
 *   - fa_lbl_softmax reads S[i][j] for visible j (j < ld otherwise unread), writes P[i][j] for every
 *     j < E (0 for masked j) and nothing else of P; P may be the same buffer as S (in place) or
 *     disjoint from it, but must not partly overlap it;
 *   - fa_lbl_pv reads P[i][j] and V rows j for j < E only (V rows j >= Sk count as zeros).
 * Causal masking and GQA as for fa_fwd_ex. Supported dimensions: d_qk in {64, 128, 192} for the
 * scores, d_v in {64, 128} for P V; Sk <= 2^22.
 *
 * Errors (host checks, in this order; on error nothing is launched): sizes as for fa_fwd_ex or
 * Sk > 2^22 (FA_ERR_BAD_SHAPE), head dimension not supported (FA_ERR_UNSUPPORTED), a NULL buffer
 * that has elements (FA_ERR_NULL_POINTER; LSE may be NULL), scale not finite (FA_ERR_BAD_SCALE), a
 * pointer not 16-byte aligned or LSE not 4-byte aligned (FA_ERR_UNSUPPORTED). B*Hq*Sq == 0 returns
 * FA_OK without a launch. Each operator enqueues one kernel on `stream`.
 */
fa_status_t fa_lbl_scores(const void* Q, const void* K, void* S, int B, int Hq, int Hkv, int Sq, int Sk,
                          int d_qk, float scale, int causal, hipStream_t stream);
fa_status_t fa_lbl_softmax(const void* S, void* P, float* LSE, int B, int Hq, int Sq, int Sk, int causal,
                           hipStream_t stream);
fa_status_t fa_lbl_pv(const void* P, const void* V, void* O, int B, int Hq, int Hkv, int Sq, int Sk, int d_v,
                      int causal, hipStream_t stream);

/* Row stride ld (elements) of the spill buffers: Sk rounded up to 64; -1 if Sk < 0 or Sk > 2^22. */
int fa_lbl_ld(int Sk);

/* Bytes of spill buffer for the whole problem, B * Hq * Sq * ld * 2; 0 if B, Hq, Sq or Sk <= 0;
 * SIZE_MAX if Sk > 2^22 or the count overflows. */
size_t fa_lbl_workspace_bytes(int B, int Hq, int Sq, int Sk);

/*
 * fa_fwd_unfused -- the three layer-by-layer operators in sequence on `stream`, producing O and
 * (optionally) LSE like fa_fwd_ex. The score matrix and then, in place, the probabilities of a
 * chunk of the problem live in `workspace` (caller-owned device memory, 16-byte aligned,
 * overwritten; not to be touched until the work on `stream` has completed). A chunk is as many whole
 * query heads as fit (a multiple of Hq / Hkv heads when more than that many fit) or, when one head
 * does not fit, as many blocks of 128 query rows of one head as fit; each chunk is three launches.
 * workspace_bytes >= fa_lbl_workspace_bytes(B, Hq, Sq, Sk) runs the whole problem as one chunk;
 * the least accepted is min(Sq, 128) * fa_lbl_ld(Sk) * 2. Supported dimensions: d_qk in
 * {64, 128, 192}, d_v in {64, 128}.
 *
 * Errors: as for the operators (sizes, head dimensions, pointers, scale, alignment of Q, K, V, O,
 * LSE), then workspace NULL or smaller than the least size (FA_ERR_WORKSPACE), then workspace not
 * 16-byte aligned (FA_ERR_UNSUPPORTED). B*Hq*Sq == 0 returns FA_OK without touching the workspace.
 * With Sk == 0 no workspace is needed and every row gets O = 0, LSE = -inf.
 */
fa_status_t fa_fwd_unfused(const void* Q, const void* K, const void* V, void* O, float* LSE, int B, int Hq,
                           int Hkv, int Sq, int Sk, int d_qk, int d_v, float scale, int causal,
                           void* workspace, size_t workspace_bytes, hipStream_t stream);

/* Static, human-readable name of a status code ("FA_OK", ...); "unknown status" otherwise. */
const char* fa_status_str(fa_status_t s);

/* Query rows per workgroup of the fused kernel's long instance for the given head dimensions when a
 * workgroup holds one query head (256); 0 if unsupported. It runs split mode, every (192, 128)
 * problem, and problems at (d_qk, d_v) = (64, 64) or (128, 128) with more such blocks
 * (B * Hq * ceil(Sq / rows)) than the other instances take (fa_fwd_rows). When Hq / Hkv is divisible
 * by 2 or 4 a workgroup holds that many query heads of one key/value head with a half or a quarter of
 * these rows each. Host arithmetic only. */
int fa_block_rows(int d_qk, int d_v, int causal);

/* Query rows per workgroup holding one query head of the fused-kernel instance that fa_fwd and
 * fa_fwd_ex (without split mode) launch for a problem of B batches, Hq query heads and Sq query rows:
 * 256 (long instance: one workgroup per compute unit), 128 (short instance: two per compute unit, at
 * most 1024 blocks at d = 64 and 256 at d = 128, i.e. blocks of the long instance's rows) or 64 (key
 * halves: each half of a workgroup's waves takes one half of every key tile, and the halves are
 * merged at the end; causal problems of at most 320 blocks at d = 64 and 192 at d = 128, others of at
 * most 64 and 128). Every instance computes the same function (Eq. (1) by Alg. 1); which one runs
 * follows from the grid size alone. 0 for unsupported head dimensions or negative sizes. Host
 * arithmetic only. */
int fa_fwd_rows(int B, int Hq, int Sq, int d_qk, int d_v, int causal);

#ifdef __cplusplus
}
#endif

#endif /* FA_MI355X_FA_H */
