/*
 * attn.h - fused scaled-dot-product attention, forward and backward, for AMD
 * Instinct MI355X (gfx950).  C ABI of libattn.so.
 *
 * What is computed (PTXBench, Appendix A, paragraph "Workloads"): the forward
 * takes bf16 Q, K, V and returns the bf16 attention output O (same shape as Q)
 * and the fp32 log-sum-exp of every query row; the backward additionally takes
 * O, its upstream gradient dO and the log-sum-exp, and returns bf16 dQ, dK,
 * dV.  Causal variants apply a lower-triangular mask: key j is visible to
 * query i iff j <= i.  Grouped-query variants ("Generalization attention
 * workloads") let Hq query heads share Hkv key/value heads: query head h reads
 * key/value head h / (Hq/Hkv), and dK, dV are summed over each group.  The
 * ragged-prefill variant packs several sequences of different lengths; no
 * attention crosses a sequence boundary and positions are local to each
 * sequence.
 *
 *   O   = softmax(scale * Q K^T + mask) V
 *   LSE = log(sum_j exp(scale * q_i . k_j))  over the visible keys j, natural
 *         log, scale included (the L_i = m_i + log l_i of the epilogue of the
 *         corrected FlashAttention-3 Algorithm 2, Appendix A)
 *
 * Layouts (all tensors contiguous, bf16 = raw IEEE bfloat16 bits):
 *   fixed length : q, o, dO, dq   [B, Hq,  S, D]     lse [B, Hq, S] fp32
 *                  k, v, dk, dv   [B, Hkv, S, D]
 *   packed       : q, o, dO, dq   [T, Hq,  D]        lse [Hq, T] fp32
 *                  k, v, dk, dv   [T, Hkv, D]
 *                  sequence s owns rows cu_seqlens[s] .. cu_seqlens[s+1]-1;
 *                  cu_seqlens is an int32 device array of nseq+1 entries,
 *                  non-decreasing, starting at 0 and ending at T.
 *
 * Ownership: every pointer is device memory owned by the caller.  Inputs are
 * read only; outputs are fully overwritten (never accumulated into).  The
 * library allocates and frees nothing; the backward's scratch space is a
 * caller-provided workspace of attn_bwd_workspace_size() bytes.
 *
 * Asynchrony: all work is enqueued on `stream` (0 = the null stream).  No
 * call synchronises or copies between host and device; the caller
 * synchronises before reading results or reusing buffers.
 *
 * Errors: every call validates its arguments on the host before touching the
 * GPU and returns ATTN_OK or a negative attn_status_t; nothing aborts.  The
 * library never reads device memory on the host, so it cannot check the
 * contents of cu_seqlens: the kernels clamp out-of-range offsets so that a
 * bad array cannot make them access memory outside the tensors, but the
 * results are then meaningless (the Python binding checks the array on the
 * host).  A problem with no rows (B == 0, S == 0, nseq == 0 or T == 0) is a
 * no-op that returns ATTN_OK; its pointers may then be null.
 */
#ifndef ATTN_H
#define ATTN_H

#include <stddef.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  ATTN_OK = 0,
  ATTN_ERR_NULL = -1,       /* a required pointer is null */
  ATTN_ERR_SHAPE = -2,      /* a size is negative, Hq/Hkv < 1, or too large
                               (S or max_seqlen > 65535*128, Hq*D > 2^22) */
  ATTN_ERR_GQA = -3,        /* Hq is not a multiple of Hkv, or (decode)
                               Hq / Hkv > 32 */
  ATTN_ERR_HEAD_DIM = -4,   /* D is not 64, 96 or 128 */
  ATTN_ERR_ALIGN = -5,      /* a pointer is not 16-byte aligned */
  ATTN_ERR_WORKSPACE = -6,  /* workspace null or smaller than required */
  ATTN_ERR_HIP = -7,        /* a kernel launch failed (hipGetLastError) */
  ATTN_ERR_VALUE = -8,      /* scale not finite or not > 0, causal not 0/1,
                               max_seqlen (max_qlen, max_kvlen) < 1, or a bad
                               backward phase mask */
  ATTN_ERR_SCRATCH = -9     /* attn_bwd_noalloc: the problem needs more than
                               ATTN_BWD_NOALLOC_SCRATCH_BYTES of scratch */
} attn_status_t;

/*
 * Forward, fixed length.  q [B,Hq,S,D], k/v [B,Hkv,S,D] in; o [B,Hq,S,D] and
 * lse [B,Hq,S] out.  causal is 0 or 1; scale is the softmax scale, finite
 * and > 0 (1/sqrt(D) in every measured workload).
 */
int attn_fwd(const void* q, const void* k, const void* v, void* o, float* lse,
             int B, int Hq, int Hkv, int S, int D, int causal, float scale,
             hipStream_t stream);

/* Bytes of backward workspace for the fixed-length layout (fp32 -Delta and
 * fp32 L log2(e), one of each per query row and head). */
size_t attn_bwd_workspace_size(int B, int Hq, int Hkv, int S, int D);

/*
 * Backward, fixed length.  Consumes q, k, v, the forward's o and lse, and
 * dO; writes dq [B,Hq,S,D] and dk, dv [B,Hkv,S,D] (dk, dv summed over each
 * query-head group).  Delta_i = sum_d dO_id * O_id (stored negated) and
 * lse_i * log2(e) are precomputed into the workspace; P is recomputed from
 * them.  The gradients are of the loss
 * sum(dO * O) with O = attention(q, k, v).  The result is deterministic
 * (no atomics).
 */
int attn_bwd(const void* q, const void* k, const void* v, const void* o,
             const float* lse, const void* dO, void* dq, void* dk, void* dv,
             int B, int Hq, int Hkv, int S, int D, int causal, float scale,
             void* workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * Backward, fixed length, for callers that cannot allocate memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc): attn_bwd without a workspace argument.  Its scratch (the
 * same fp32 -Delta and L log2(e) arrays) is a device array inside the
 * library of ATTN_BWD_NOALLOC_SCRATCH_BYTES, which every GPU the library
 * runs on holds until the process ends; the call itself allocates nothing.
 * A problem whose attn_bwd_workspace_size exceeds it (B * Hq * S above
 * 2,097,152) returns ATTN_ERR_SCRATCH before any GPU work.  Every call on
 * one GPU uses that GPU's one scratch array: calls that can overlap on a
 * GPU (other streams, other host threads) race and must be ordered by the
 * caller.  The first call on a device looks up the array's address there
 * (hipGetSymbolAddress, with that device made current for the lookup).
 * Arguments, layouts, results and errors otherwise as for attn_bwd; the
 * results are bitwise equal to attn_bwd's.
 */
#define ATTN_BWD_NOALLOC_SCRATCH_BYTES (16u << 20)
int attn_bwd_noalloc(const void* q, const void* k, const void* v, const void* o,
                     const float* lse, const void* dO, void* dq, void* dk, void* dv,
                     int B, int Hq, int Hkv, int S, int D, int causal, float scale,
                     hipStream_t stream);

/*
 * Forward, packed variable length (ragged prefill).  total = T rows;
 * max_seqlen >= the longest sequence (it sizes the launch; a longer sequence
 * is processed only up to max_seqlen rows).
 */
int attn_fwd_varlen(const void* q, const void* k, const void* v, void* o,
                    float* lse, const int* cu_seqlens, int nseq,
                    int max_seqlen, int total, int Hq, int Hkv, int D,
                    int causal, float scale, hipStream_t stream);

/* Bytes of backward workspace for the packed layout (fp32 -Delta and fp32
 * L log2(e), one of each per query row and head). */
size_t attn_bwd_varlen_workspace_size(int total, int Hq, int Hkv, int D);

/* Backward, packed variable length.  Same contract as attn_bwd. */
int attn_bwd_varlen(const void* q, const void* k, const void* v,
                    const void* o, const float* lse, const void* dO, void* dq,
                    void* dk, void* dv, const int* cu_seqlens, int nseq,
                    int max_seqlen, int total, int Hq, int Hkv, int D,
                    int causal, float scale, void* workspace,
                    size_t workspace_bytes, hipStream_t stream);

/*
 * The backward in separately enqueued phases, for callers that time or
 * schedule its two kernels on their own.  `phases` is a bit mask:
 *   ATTN_BWD_DQ   computes -Delta and lse * log2(e) into the workspace,
 *                 then dq;
 *   ATTN_BWD_DKDV computes dk and dv from the workspace of an ATTN_BWD_DQ phase
 *                 enqueued earlier on the same stream with the same
 *                 workspace and inputs.
 * phases = ATTN_BWD_DQ | ATTN_BWD_DKDV is exactly attn_bwd / attn_bwd_varlen.
 * With ATTN_BWD_DKDV, one of the two bits below may be added to choose the
 * form of the dk/dv kernel at D = 96 and 128 (for tests and tuning; D = 64
 * has only the second form and ignores them):
 *   ATTN_BWD_DKDV_ONE_PER_CU  eight wavefronts per 128 keys, one workgroup
 *                             per CU;
 *   ATTN_BWD_DKDV_TWO_PER_CU  four wavefronts per 128 keys, two (at D = 64
 *                             three) per CU.
 * Both give dk and dv equal up to the order of floating-point additions.
 * Without either the library picks two per CU, unless the mask is causal
 * and there are fewer than 1,024 blocks of 128 keys (all workgroups would
 * then be resident at once, and the causal blocks' unequal work could not
 * be balanced).  Any other value returns ATTN_ERR_VALUE.  Arguments are as
 * for attn_bwd / attn_bwd_varlen.
 */
#define ATTN_BWD_DQ 1
#define ATTN_BWD_DKDV 2
#define ATTN_BWD_DKDV_ONE_PER_CU 4
#define ATTN_BWD_DKDV_TWO_PER_CU 8

/* The dk/dv form attn_bwd (packed 0: nseg = B, S the sequence length) or
 * attn_bwd_varlen (packed 1: nseg = nseq, S = max_seqlen, total) picks for
 * these arguments: ATTN_BWD_DKDV_ONE_PER_CU or ATTN_BWD_DKDV_TWO_PER_CU
 * (always the latter at D = 64); a negative status for bad arguments.  No
 * GPU call. */
int attn_bwd_dkdv_form(int nseg, int Hkv, int S, int total, int D, int causal, int packed);
int attn_bwd_phases(const void* q, const void* k, const void* v, const void* o,
                    const float* lse, const void* dO, void* dq, void* dk,
                    void* dv, int B, int Hq, int Hkv, int S, int D, int causal,
                    float scale, void* workspace, size_t workspace_bytes,
                    int phases, hipStream_t stream);
int attn_bwd_varlen_phases(const void* q, const void* k, const void* v,
                           const void* o, const float* lse, const void* dO,
                           void* dq, void* dk, void* dv,
                           const int* cu_seqlens, int nseq, int max_seqlen,
                           int total, int Hq, int Hkv, int D, int causal,
                           float scale, void* workspace,
                           size_t workspace_bytes, int phases,
                           hipStream_t stream);

/*
 * Paged key/value cache, page size 1 (the paged causal prefill and paged
 * decode workloads of PTXBench, Appendix A, "Generalization attention
 * workloads"; forward only, as there).
 *
 *   k_cache, v_cache  [num_pages, Hkv, D] bf16: one token per page.
 *   kv_indptr         int32 [batch+1], non-decreasing, from 0 to nnz.
 *   kv_indices        int32 [nnz]: request b's keys and values are the pages
 *                     kv_indices[kv_indptr[b]] .. kv_indices[kv_indptr[b+1]-1],
 *                     in that order (kv_len_b of them).
 *
 * Attention of each request's queries over its keys, as for the packed
 * layout.  When a request has q_len queries and kv_len keys, its queries are
 * the last q_len of its kv_len positions: with the causal mask, query i
 * (0-based within the request) sees keys j <= i + kv_len - q_len (the
 * lower-triangular mask when q_len == kv_len).  Rows that see no key get
 * O = 0 and lse = -inf.
 *
 * The library reads the index arrays only on the device: offsets are clamped
 * into [0, nnz] and a page number outside [0, num_pages) reads as a zero key
 * and value row, so bad contents cannot make a kernel access memory outside
 * the given arrays (the results are then meaningless; the Python binding
 * checks the arrays on the host).  num_pages * Hkv * D * 2 must be below
 * 2^31 and nnz at most 2^29 (ATTN_ERR_SHAPE).  The index arrays need 4-byte
 * alignment, every other pointer 16-byte alignment.
 */

/* Bytes of workspace for attn_fwd_paged: 0 when the prefill runs unsplit
 * (its unsplit grid of a workgroup per 128-query block, per request and
 * query head, fills at least half of the 256 CUs of the MI355X, or no
 * request is longer than 256 keys), else the partial results of the
 * 256-key chunks: fp32 [total_q, Hq, ceil(max_kvlen / 256), D + 1], rounded
 * up.  The size depends on the arguments alone. */
size_t attn_fwd_paged_workspace_size(int batch, int max_qlen, int total_q, int max_kvlen,
                                     int Hq, int Hkv, int D);

/* The form attn_fwd_paged runs for these arguments (with_workspace 1: a
 * workspace of attn_fwd_paged_workspace_size bytes is passed; 0: none).  No
 * GPU call.
 *   ATTN_FWD_PAGED_UNSPLIT     one 4-wavefront workgroup per 128-query block
 *                              (the unsplit grid fills the 256 CUs);
 *   ATTN_FWD_PAGED_KEY_HALVES  one 8-wavefront workgroup per block, whose two
 *                              halves take alternate key tiles and combine on
 *                              chip (an unsplit grid of fewer workgroups than
 *                              CUs);
 *   ATTN_FWD_PAGED_SPLIT       256-key chunks, one workgroup each, then a merge
 *                              kernel (a workspace, a request longer than 256
 *                              keys, and an unsplit grid of fewer than 128
 *                              workgroups).
 * Returns ATTN_ERR_SHAPE for batch, max_qlen or Hq below 1, max_kvlen below
 * 0 or batch * Hq above 2^30, ATTN_ERR_VALUE for another with_workspace. */
#define ATTN_FWD_PAGED_UNSPLIT 0
#define ATTN_FWD_PAGED_KEY_HALVES 1
#define ATTN_FWD_PAGED_SPLIT 2
int attn_fwd_paged_form(int batch, int max_qlen, int max_kvlen, int Hq, int with_workspace);

/*
 * Paged prefill.  q, o [total_q, Hq, D] packed by qo_indptr (int32 [batch+1],
 * from 0 to total_q, as cu_seqlens); lse [Hq, total_q] fp32.  max_qlen >= the
 * longest query run (it sizes the launch).  max_kvlen >= the largest key
 * count of a request (keys past it are ignored).  causal 0 or 1.
 *
 * An unsplit grid with fewer workgroups than CUs runs two halves of each
 * workgroup over alternate key tiles, combined on chip.  When
 * attn_fwd_paged_workspace_size is not 0 and a workspace is given (at least
 * that many bytes, 16-byte aligned, caller-owned, contents irrelevant), the
 * keys of every query block are split into chunks of 256, one workgroup
 * each, and a second kernel merges the chunks' partial results, so that a
 * few long requests still fill the device.  With a null workspace the
 * prefill runs unsplit (a non-null one that is too small is
 * ATTN_ERR_WORKSPACE).  Calls that share a workspace must not overlap.
 */
int attn_fwd_paged(const void* q, const void* k_cache, const void* v_cache, void* o,
                   float* lse, const int* qo_indptr, const int* kv_indptr,
                   const int* kv_indices, int batch, int max_qlen, int total_q, int max_kvlen,
                   int nnz, int num_pages, int Hq, int Hkv, int D, int causal, float scale,
                   void* workspace, size_t workspace_bytes, hipStream_t stream);

/* Bytes of workspace for attn_decode_paged (partial outputs of the key
 * chunks: fp32 [batch, Hq, ceil(max_kvlen / 64), D + 1], rounded up). */
size_t attn_decode_paged_workspace_size(int batch, int max_kvlen, int Hq, int Hkv, int D);

/*
 * Paged decode: one query per request.  q, o [batch, Hq, D]; lse [Hq, batch]
 * fp32.  Every key of the request is visible.  max_kvlen >= the longest
 * request (it sizes the launch and the workspace; a longer request is
 * truncated to its first max_kvlen keys).  Hq / Hkv must be at most 32
 * (ATTN_ERR_GQA).  The workspace (16-byte aligned, caller-owned, contents
 * irrelevant) holds the partial results of the key chunks; calls that share
 * a workspace must not overlap.  A request with no keys gets O = 0 and
 * lse = -inf.
 */
int attn_decode_paged(const void* q, const void* k_cache, const void* v_cache, void* o,
                      float* lse, const int* kv_indptr, const int* kv_indices, int batch,
                      int max_kvlen, int nnz, int num_pages, int Hq, int Hkv, int D,
                      float scale, void* workspace, size_t workspace_bytes,
                      hipStream_t stream);

/*
 * The decode in separately enqueued phases, for callers that time or
 * schedule its two kernels on their own.  `phases` is a bit mask:
 *   ATTN_DECODE_SPLIT  per-chunk partial results (and the final result of
 *                      requests with at most 64 keys);
 *   ATTN_DECODE_MERGE  the merge of the chunks of every longer request (and
 *                      the result of requests with no keys), reading the
 *                      workspace of an ATTN_DECODE_SPLIT phase enqueued
 *                      earlier on the same stream with the same arguments.
 * Both bits together are exactly attn_decode_paged; any other value returns
 * ATTN_ERR_VALUE.
 */
#define ATTN_DECODE_SPLIT 1
#define ATTN_DECODE_MERGE 2
int attn_decode_paged_phases(const void* q, const void* k_cache, const void* v_cache, void* o,
                             float* lse, const int* kv_indptr, const int* kv_indices,
                             int batch, int max_kvlen, int nnz, int num_pages, int Hq,
                             int Hkv, int D, float scale, void* workspace,
                             size_t workspace_bytes, int phases, hipStream_t stream);

/*
 * BF16 GEMM C = A B^T (the fifth primary workload of PTXBench, Appendix A,
 * "Workloads": A 8192 x 5120, B 7168 x 5120, C 8192 x 7168).  a [M, K],
 * b [N, K], c [M, N], all row-major bf16 and 16-byte aligned; fp32
 * accumulation, C rounded to bf16 (round to nearest even).  K and N must be
 * multiples of 8 and K * 512 below 2^31 (ATTN_ERR_SHAPE); M is free.
 * K == 0 gives C = 0 (a and b may then be null); M == 0 or N == 0 is a
 * no-op (every pointer may then be null).
 * Ownership, asynchrony and errors as for the attention calls.
 */
int attn_gemm_bf16_nt(const void* a, const void* b, void* c, int M, int N, int K,
                      hipStream_t stream);

/* Static, human-readable text for a status code (never null). */
const char* attn_status_string(int status);

#ifdef __cplusplus
}
#endif

#endif /* ATTN_H */
