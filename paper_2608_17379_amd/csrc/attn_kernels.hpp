// Internal interface between the C ABI (attn_api.cpp) and the HIP kernels.
//
// A "segment" is one batch entry (fixed length) or one packed sequence.  Row i
// of head h of segment z of a q-like tensor (q, o, dO, dq; Hq heads) is at
//   base + start * row_stride + z * batch_stride + h * head_stride
//        + i * row_stride                                    (elements)
// where start = cu[z] and batch_stride = 0 for packed input, and start = 0
// for fixed-length input;
// k-like tensors (k, v, dk, dv; Hkv heads) use the kv strides.  Row-indexed
// fp32 arrays (lse, Delta) follow the same rule with their own strides and a
// unit row stride.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace attn {

// Order of the workgroups of a launch over (block, head): the hardware
// deals workgroup ids to the chip's eight XCDs in turn (id % 8), and each XCD
// has its own L2.  Workgroup id L is given to kv-head group
// gk = L % 8 + 8 i (a segment's kv head with its G query heads, or G = 1 for
// a launch over kv heads), so that every workgroup reading one K/V head (or
// one group's Q and dO) runs on one XCD.  Within an XCD (ids L / 8 in
// dispatch order) the groups come in windows of W: a window's blocks go
// heaviest first (p = 0 has the most work under the causal mask), each
// block for all the window's groups and their G heads side by side.  W = 1
// (one group at a time) keeps the workgroups resident at a time on a few
// heads' tiles in the L2; a causal launch takes windows of at least 256
// workgroups, so that its heavy blocks are still dispatched before the
// light ones (a window's last heavy block would otherwise start late).
constexpr int kXcds = 8;
struct XcdOrder {
  int nkv;       // groups: segments x Hkv
  int G;         // heads per group
  int nb;        // blocks per head (the grid's extent; a segment may have fewer)
  int per_xcd;   // groups per XCD: ceil(nkv / 8)
  int W;         // groups per window
};
inline XcdOrder xcd_order(int nseg, int Hkv, int G, int nb, bool causal) {
  const int nkv = nseg * Hkv;
  const int per = (nkv + kXcds - 1) / kXcds;
  int W = 1;
  if (causal) {
    const int64_t per_group = (int64_t)nb * G;
    W = (int)((256 + per_group - 1) / per_group);
  }
  W = W < 1 ? 1 : (W > per ? per : W);
  return XcdOrder{nkv, G, nb, per, W};
}
// Workgroups of such a launch (the last XCDs' unused slots exit at once).
inline int64_t xcd_grid(const XcdOrder& o) {
  return (int64_t)kXcds * o.per_xcd * o.G * o.nb;
}
// Workgroup L's group gk, head j within the group and block index p; false
// for an unused slot.
__device__ __forceinline__ bool xcd_decode(int L, const XcdOrder& o, int& gk, int& j, int& p) {
  const int r = L % kXcds;
  int s = L / kXcds;
  const int full = o.W * o.nb * o.G;          // workgroups of a whole window
  const int w = s / full;                     // window (the last may be short)
  s -= w * full;
  const int wl = min(o.W, o.per_xcd - w * o.W);   // groups in this window
  const int per_block = wl * o.G;
  p = s / per_block;
  s -= p * per_block;
  const int ig = s / o.G;
  j = s - ig * o.G;
  gk = r + kXcds * (w * o.W + ig);
  return gk < o.nkv;
}

struct Layout {
  const int* cu;           // packed: cu_seqlens (device); fixed: nullptr
  int S;                   // fixed: sequence length; packed: max_seqlen
  int total;               // packed: T (rows); fixed: unused
  int nseg;                // B or nseq
  int Hq, Hkv, group;      // group = Hq / Hkv
  int64_t q_batch, q_head, q_row;     // strides of q-like tensors
  int64_t kv_batch, kv_head, kv_row;  // strides of k-like tensors
  int64_t r_batch, r_head;            // strides of lse / Delta (row stride 1)
  // Paged key/value cache (page size 1), forward only; kv_cu == nullptr
  // otherwise.  Keys of segment z are the cache rows kv_idx[kv_cu[z]] ..
  // kv_idx[kv_cu[z+1]-1], each kv_row elements apart (k-like strides with
  // kv_batch = 0 and start 0); the segment's queries are the last of its
  // key positions.
  const int* kv_cu;        // [nseg + 1] offsets into kv_idx (device)
  const int* kv_idx;       // [nnz] page numbers (device)
  int nnz;                 // entries of kv_idx
  int num_pages;           // rows of the cache
};

struct FwdArgs {
  Layout L;
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  uint16_t* o;
  float* lse;
  float scale_log2;        // softmax scale * log2(e)
  int causal;
  // Paged prefill only.  Keys of a request past max_kvlen are ignored.  With
  // split > 0 the keys of every query block are cut into chunks of `split`
  // keys (a multiple of 128), one workgroup each: a block with more than one
  // chunk writes normalised partial outputs and base-2 log-sum-exps to the
  // workspace, which fwd_merge_kernel combines.
  int max_kvlen;
  int split;               // keys per chunk, or 0 (unsplit)
  int nsplit;              // chunk slots per (query row, head): the grid's z extent
  float* part_o;           // workspace [total_q, Hq, nsplit, D] fp32
  float* part_lse;         // workspace [total_q, Hq, nsplit] fp32, log2 units
  XcdOrder xo;             // unpaged: workgroup order (set by the launcher)
};

struct BwdArgs {
  Layout L;
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  const uint16_t* o;
  const float* lse;
  const uint16_t* dout;
  uint16_t* dq;
  uint16_t* dk;
  uint16_t* dv;
  float* delta;            // workspace: Delta, same layout as lse
  float* lse2;             // workspace: lse * log2(e), same layout as lse
  float scale;             // softmax scale
  float scale_log2;        // scale * log2(e)
  int causal;
  int dkdv_form;           // D = 96, 128: 0 chosen by the grid, 1 one, 2 two workgroups per CU
  XcdOrder xo;             // dQ kernel's workgroup order (set by the launcher)
  XcdOrder xk;             // dK/dV kernel's workgroup order (G = 1: kv heads)
};

// Paged decode: one query row per request (q, o [batch, Hq, D], lse
// [Hq, batch]) against its pages, split into chunks of keys whose partial
// results go to the workspace and are merged by a second kernel.
struct DecodeArgs {
  const uint16_t* q;
  const uint16_t* k;       // cache [num_pages, Hkv, D]
  const uint16_t* v;
  uint16_t* o;
  float* lse;
  const int* kv_cu;        // [batch + 1]
  const int* kv_idx;       // [nnz]
  int batch, Hq, Hkv, group, nnz, num_pages, max_kvlen;
  int nchunk;              // key chunks per request (max_kvlen rounded up)
  float scale_log2;        // softmax scale * log2(e)
  float* part_o;           // workspace [batch, Hq, nchunk, D] fp32
  float* part_lse;         // workspace [batch, Hq, nchunk] fp32, log2 units
};

// BF16 GEMM C = A B^T: A [M, K], B [N, K], C [M, N], row-major, K % 8 == 0,
// N % 8 == 0; tiles of 256 x 256.
struct GemmArgs {
  const uint16_t* a;
  const uint16_t* b;
  uint16_t* c;
  int M, N, K;
  int tiles_m, tiles_n;
  int tile0;               // first tile of a launch (set by the launcher)
};

// Launchers: enqueue on `stream`, return the hipGetLastError() of the launch.
// cus: compute units of the device (sizes the rounds of workgroups).
hipError_t launch_gemm(const GemmArgs& g, int cus, hipStream_t stream);
hipError_t launch_fwd(const FwdArgs& a, int D, hipStream_t stream);
// Keys per chunk of the decode split (sizes the workspace).
constexpr int kDecodeChunk = 64;
constexpr int kChipCUs = 256;        // compute units of the MI355X
constexpr int kFwdSplitKeys = 256;   // keys per chunk of a split paged prefill
constexpr int kFwdBlockRows = 128;   // query rows per forward workgroup

// An unsplit paged prefill runs the forward's 8-wavefront key-halves form
// when its grid (a workgroup per 128-query block, per request and query
// head: `heads` = requests x query heads) has fewer workgroups than the
// chip has CUs.
inline bool paged_key_halves(int64_t heads, int max_qlen) {
  return heads * ((max_qlen + kFwdBlockRows - 1) / kFwdBlockRows) < kChipCUs;
}
// phases: bit 0 = split kernel, bit 1 = merge kernel.
hipError_t launch_decode(const DecodeArgs& a, int D, int phases, hipStream_t stream);
// phases: bit 0 = Delta and dQ kernel, bit 1 = dK/dV kernel.
hipError_t launch_bwd(const BwdArgs& a, int D, int phases, hipStream_t stream);
// The dK/dV form launch_bwd picks when BwdArgs::dkdv_form is 0: 1 (eight
// wavefronts, one workgroup per CU) or 2 (four wavefronts, two per CU);
// always 2 at D = 64.
int dkdv_form_for(int nseg, int Hkv, int S, int total, bool packed, int D, bool causal);

}  // namespace attn
