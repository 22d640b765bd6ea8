// C ABI of libattn.so: host-side validation, layout description and launch.
// No call here reads device memory, allocates, copies or synchronises.
#include <math.h>
#include <stdint.h>

#include <atomic>
#include <initializer_list>
#include <mutex>

#include "../../include/attn.h"
#include "attn_kernels.hpp"

namespace {

using attn::Layout;

constexpr int64_t kMaxGridY = 65535;              // launch rows of tiles (128 rows each)

bool misaligned(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) != 0; }

// Shared checks of the scalar arguments.  Returns ATTN_OK or an error.
int check_common(int Hq, int Hkv, int D, int causal, float scale) {
  if (Hq < 1 || Hkv < 1) return ATTN_ERR_SHAPE;
  if (Hq % Hkv != 0) return ATTN_ERR_GQA;
  if (D != 64 && D != 96 && D != 128) return ATTN_ERR_HEAD_DIM;
  // Bytes of 128 rows of one packed tensor must fit the 31-bit offsets of
  // the kernels' buffer loads.
  if ((int64_t)Hq * D * 2 * 128 > 0x7fffffff) return ATTN_ERR_SHAPE;
  if (causal != 0 && causal != 1) return ATTN_ERR_VALUE;
  // The kernels take row maxima of the raw scores, so the scale must be > 0.
  if (!(scale > 0.f) || !isfinite(scale)) return ATTN_ERR_VALUE;
  return ATTN_OK;
}

int check_rows(int64_t rows) {
  if (rows < 0) return ATTN_ERR_SHAPE;
  if (rows > kMaxGridY * 128) return ATTN_ERR_SHAPE;
  return ATTN_OK;
}

Layout fixed_layout(int B, int Hq, int Hkv, int S, int D) {
  Layout L{};
  L.cu = nullptr;
  L.S = S;
  L.total = 0;
  L.nseg = B;
  L.Hq = Hq;
  L.Hkv = Hkv;
  L.group = Hq / Hkv;
  L.q_row = D;
  L.q_head = (int64_t)S * D;
  L.q_batch = (int64_t)Hq * S * D;
  L.kv_row = D;
  L.kv_head = (int64_t)S * D;
  L.kv_batch = (int64_t)Hkv * S * D;
  L.r_head = S;
  L.r_batch = (int64_t)Hq * S;
  return L;
}

Layout packed_layout(const int* cu, int nseq, int max_seqlen, int total, int Hq, int Hkv, int D) {
  Layout L{};
  L.cu = cu;
  L.S = max_seqlen;
  L.total = total;
  L.nseg = nseq;
  L.Hq = Hq;
  L.Hkv = Hkv;
  L.group = Hq / Hkv;
  L.q_row = (int64_t)Hq * D;
  L.q_head = D;
  L.q_batch = 0;
  L.kv_row = (int64_t)Hkv * D;
  L.kv_head = D;
  L.kv_batch = 0;
  L.r_head = total;
  L.r_batch = 0;
  return L;
}

// The attention kernels run 1-D grids over (block of 128 rows, head) in the
// XCD-aware order; the largest (query heads) must fit a launch.
bool grid_too_large(int64_t nseg, int Hq, int Hkv, int64_t rows) {
  const int64_t nkv = nseg * Hkv;
  const int64_t n = (int64_t)attn::kXcds * ((nkv + attn::kXcds - 1) / attn::kXcds) * (Hq / Hkv) *
                    ((rows + 127) / 128);
  return n > 0x7fffffff;
}

bool any_null(std::initializer_list<const void*> ps) {
  for (const void* p : ps)
    if (!p) return true;
  return false;
}

bool any_misaligned(std::initializer_list<const void*> ps) {
  for (const void* p : ps)
    if (misaligned(p)) return true;
  return false;
}

// Key split of a paged prefill (see attn::FwdArgs).
struct PagedSplit {
  int max_kvlen;
  int split;
  int nsplit;
  float* part_o;
  float* part_lse;
};

int fwd_common(const void* q, const void* k, const void* v, void* o, float* lse,
               const Layout& L, int D, int causal, float scale, hipStream_t stream,
               const PagedSplit* ps = nullptr) {
  if (any_null({q, k, v, o, lse})) return ATTN_ERR_NULL;
  if (any_misaligned({q, k, v, o, lse})) return ATTN_ERR_ALIGN;
  attn::FwdArgs a{};
  if (ps) {
    a.max_kvlen = ps->max_kvlen;
    a.split = ps->split;
    a.nsplit = ps->nsplit;
    a.part_o = ps->part_o;
    a.part_lse = ps->part_lse;
  }
  a.L = L;
  a.q = static_cast<const uint16_t*>(q);
  a.k = static_cast<const uint16_t*>(k);
  a.v = static_cast<const uint16_t*>(v);
  a.o = static_cast<uint16_t*>(o);
  a.lse = lse;
  a.scale_log2 = scale * 1.4426950408889634f;
  a.causal = causal;
  return attn::launch_fwd(a, D, stream) == hipSuccess ? ATTN_OK : ATTN_ERR_HIP;
}

// A backward phase mask: at least one kernel, and at most one dK/dV form
// bit, given only with the dK/dV phase.
bool valid_bwd_phases(int phases) {
  if (phases < 1 || phases > 15 || (phases & 3) == 0) return false;
  const int form = phases & (ATTN_BWD_DKDV_ONE_PER_CU | ATTN_BWD_DKDV_TWO_PER_CU);
  if (form == (ATTN_BWD_DKDV_ONE_PER_CU | ATTN_BWD_DKDV_TWO_PER_CU)) return false;
  return form == 0 || (phases & ATTN_BWD_DKDV) != 0;
}

int bwd_common(const void* q, const void* k, const void* v, const void* o, const float* lse,
               const void* dO, void* dq, void* dk, void* dv, const Layout& L, int D, int causal,
               float scale, void* ws, size_t ws_bytes, size_t ws_need, int phases,
               hipStream_t stream) {
  if (!valid_bwd_phases(phases)) return ATTN_ERR_VALUE;
  if (any_null({q, k, v, o, lse, dO, dq, dk, dv})) return ATTN_ERR_NULL;
  if (any_misaligned({q, k, v, o, lse, dO, dq, dk, dv})) return ATTN_ERR_ALIGN;
  if (!ws || ws_bytes < ws_need) return ATTN_ERR_WORKSPACE;
  if (misaligned(ws)) return ATTN_ERR_ALIGN;
  attn::BwdArgs a{};
  a.L = L;
  a.q = static_cast<const uint16_t*>(q);
  a.k = static_cast<const uint16_t*>(k);
  a.v = static_cast<const uint16_t*>(v);
  a.o = static_cast<const uint16_t*>(o);
  a.lse = lse;
  a.dout = static_cast<const uint16_t*>(dO);
  a.dq = static_cast<uint16_t*>(dq);
  a.dk = static_cast<uint16_t*>(dk);
  a.dv = static_cast<uint16_t*>(dv);
  a.delta = static_cast<float*>(ws);
  a.lse2 = reinterpret_cast<float*>(static_cast<char*>(ws) + ws_need / 2);
  a.scale = scale;
  a.scale_log2 = scale * 1.4426950408889634f;
  a.causal = causal;
  a.dkdv_form = (phases & ATTN_BWD_DKDV_ONE_PER_CU) ? 1 : (phases & ATTN_BWD_DKDV_TWO_PER_CU) ? 2 : 0;
  return attn::launch_bwd(a, D, phases & 3, stream) == hipSuccess ? ATTN_OK : ATTN_ERR_HIP;
}

// A paged cache must be addressable with 31-bit byte offsets from the start
// of any head's first row, and its page-index array with 31-bit offsets.
int check_cache(int num_pages, int nnz, int Hkv, int D) {
  if (num_pages < 0 || nnz < 0 || nnz > (1 << 29)) return ATTN_ERR_SHAPE;
  if ((int64_t)num_pages * Hkv * D * 2 > 0x7fffffff) return ATTN_ERR_SHAPE;
  return ATTN_OK;
}

bool misaligned4(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 3u) != 0; }

int64_t decode_chunks(int max_kvlen) {
  return ((int64_t)max_kvlen + attn::kDecodeChunk - 1) / attn::kDecodeChunk;
}

size_t round256(int64_t bytes) { return (size_t)((bytes + 255) / 256 * 256); }

// A paged prefill whose unsplit grid (a workgroup per 128-row query block,
// per request and query head) has fewer workgroups than the MI355X has CUs
// runs the forward's key-halves form, one 8-wavefront workgroup per CU;
// when even that leaves more than half the CUs idle, it is split into
// chunks of keys instead, when its requests are longer than one chunk.  The
// rule uses the part's CU count, not a device query, so that the workspace
// size depends on the shapes alone.
using attn::kChipCUs;

int paged_split(int batch, int max_qlen, int max_kvlen, int Hq) {
  const int64_t nqt = ((int64_t)max_qlen + attn::kFwdBlockRows - 1) / attn::kFwdBlockRows;
  const int64_t wgs = (int64_t)batch * Hq * nqt;
  if (max_kvlen <= attn::kFwdSplitKeys || wgs >= kChipCUs / 2) return 0;
  return attn::kFwdSplitKeys;
}

size_t delta_bytes(int64_t rows_times_heads) {
  // fp32 Delta and fp32 L log2(e) per (row, query head), each array rounded
  // up to 256 bytes.
  return 2 * (size_t)((rows_times_heads * 4 + 255) / 256 * 256);
}

// ---------------------------------------------------------------------------
// Scratch of attn_bwd_noalloc: the backward's Delta and L log2(e) arrays in a
// file-scope device array instead of a caller workspace.  Each GPU the
// library runs on holds its own copy until the process ends.  Host code
// never passes the array's name to a kernel (on the host it only stands for
// the device symbol): the device address comes from hipGetSymbolAddress,
// taken once per device with that device current, and is kept per device.
// ---------------------------------------------------------------------------
constexpr int kMaxDevices = 64;
std::atomic<void*> g_scratch_ptr[kMaxDevices];
std::mutex g_scratch_mu;

}  // namespace

static __device__ __align__(256) unsigned char scratch[ATTN_BWD_NOALLOC_SCRATCH_BYTES];

namespace {

// Device address of `scratch` on the device `stream` belongs to.
int scratch_for(hipStream_t stream, void** out) {
  hipDevice_t dev = 0;
  if (hipStreamGetDevice(stream, &dev) != hipSuccess) return ATTN_ERR_HIP;
  if (dev < 0 || dev >= kMaxDevices) return ATTN_ERR_HIP;
  void* p = g_scratch_ptr[dev].load(std::memory_order_acquire);
  if (!p) {
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    p = g_scratch_ptr[dev].load(std::memory_order_relaxed);
    if (!p) {
      int cur = 0;
      if (hipGetDevice(&cur) != hipSuccess) return ATTN_ERR_HIP;
      if (cur != dev && hipSetDevice(dev) != hipSuccess) return ATTN_ERR_HIP;
      const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
      if (cur != dev && hipSetDevice(cur) != hipSuccess) return ATTN_ERR_HIP;
      if (e != hipSuccess || !p) return ATTN_ERR_HIP;
      g_scratch_ptr[dev].store(p, std::memory_order_release);
    }
  }
  *out = p;
  return ATTN_OK;
}

}  // namespace

extern "C" {

int attn_fwd(const void* q, const void* k, const void* v, void* o, float* lse, int B, int Hq,
             int Hkv, int S, int D, int causal, float scale, hipStream_t stream) {
  int st = check_common(Hq, Hkv, D, causal, scale);
  if (st != ATTN_OK) return st;
  if (B < 0 || (st = check_rows(S)) != ATTN_OK) return ATTN_ERR_SHAPE;
  if ((int64_t)B * Hq > (int64_t)1 << 30) return ATTN_ERR_SHAPE;
  if (grid_too_large(B, Hq, Hkv, S)) return ATTN_ERR_SHAPE;
  if (B == 0 || S == 0) return ATTN_OK;
  return fwd_common(q, k, v, o, lse, fixed_layout(B, Hq, Hkv, S, D), D, causal, scale, stream);
}

size_t attn_bwd_workspace_size(int B, int Hq, int Hkv, int S, int D) {
  (void)Hkv;
  (void)D;
  if (B <= 0 || Hq <= 0 || S <= 0) return 0;
  return delta_bytes((int64_t)B * Hq * S);
}

int attn_bwd_dkdv_form(int nseg, int Hkv, int S, int total, int D, int causal, int packed) {
  if (nseg < 0 || Hkv < 1 || S < 0 || total < 0) return ATTN_ERR_SHAPE;
  if (D != 64 && D != 96 && D != 128) return ATTN_ERR_HEAD_DIM;
  if ((causal != 0 && causal != 1) || (packed != 0 && packed != 1)) return ATTN_ERR_VALUE;
  return attn::dkdv_form_for(nseg, Hkv, S, total, packed != 0, D, causal != 0) == 1
             ? ATTN_BWD_DKDV_ONE_PER_CU
             : ATTN_BWD_DKDV_TWO_PER_CU;
}

int attn_bwd_phases(const void* q, const void* k, const void* v, const void* o, const float* lse,
                    const void* dO, void* dq, void* dk, void* dv, int B, int Hq, int Hkv, int S,
                    int D, int causal, float scale, void* workspace, size_t workspace_bytes,
                    int phases, hipStream_t stream) {
  int st = check_common(Hq, Hkv, D, causal, scale);
  if (st != ATTN_OK) return st;
  if (B < 0 || check_rows(S) != ATTN_OK) return ATTN_ERR_SHAPE;
  if ((int64_t)B * Hq > (int64_t)1 << 30) return ATTN_ERR_SHAPE;
  if (grid_too_large(B, Hq, Hkv, S)) return ATTN_ERR_SHAPE;
  if (!valid_bwd_phases(phases)) return ATTN_ERR_VALUE;
  if (B == 0 || S == 0) return ATTN_OK;
  return bwd_common(q, k, v, o, lse, dO, dq, dk, dv, fixed_layout(B, Hq, Hkv, S, D), D, causal,
                    scale, workspace, workspace_bytes, attn_bwd_workspace_size(B, Hq, Hkv, S, D),
                    phases, stream);
}

int attn_bwd(const void* q, const void* k, const void* v, const void* o, const float* lse,
             const void* dO, void* dq, void* dk, void* dv, int B, int Hq, int Hkv, int S, int D,
             int causal, float scale, void* workspace, size_t workspace_bytes,
             hipStream_t stream) {
  return attn_bwd_phases(q, k, v, o, lse, dO, dq, dk, dv, B, Hq, Hkv, S, D, causal, scale,
                         workspace, workspace_bytes, ATTN_BWD_DQ | ATTN_BWD_DKDV, stream);
}

int attn_bwd_noalloc(const void* q, const void* k, const void* v, const void* o,
                     const float* lse, const void* dO, void* dq, void* dk, void* dv, int B,
                     int Hq, int Hkv, int S, int D, int causal, float scale,
                     hipStream_t stream) {
  int st = check_common(Hq, Hkv, D, causal, scale);
  if (st != ATTN_OK) return st;
  if (B < 0 || check_rows(S) != ATTN_OK) return ATTN_ERR_SHAPE;
  if ((int64_t)B * Hq > (int64_t)1 << 30) return ATTN_ERR_SHAPE;
  if (grid_too_large(B, Hq, Hkv, S)) return ATTN_ERR_SHAPE;
  if (B == 0 || S == 0) return ATTN_OK;
  const size_t need = attn_bwd_workspace_size(B, Hq, Hkv, S, D);
  if (need > ATTN_BWD_NOALLOC_SCRATCH_BYTES) return ATTN_ERR_SCRATCH;
  if (any_null({q, k, v, o, lse, dO, dq, dk, dv})) return ATTN_ERR_NULL;
  if (any_misaligned({q, k, v, o, lse, dO, dq, dk, dv})) return ATTN_ERR_ALIGN;
  void* ws = nullptr;
  if ((st = scratch_for(stream, &ws)) != ATTN_OK) return st;
  // The dQ kernel writes Delta and L log2(e) of every row before the dK/dV
  // kernel reads them (rows past a segment end are never read), so the
  // scratch needs no clearing between calls.
  return bwd_common(q, k, v, o, lse, dO, dq, dk, dv, fixed_layout(B, Hq, Hkv, S, D), D, causal,
                    scale, ws, ATTN_BWD_NOALLOC_SCRATCH_BYTES, need,
                    ATTN_BWD_DQ | ATTN_BWD_DKDV, stream);
}

int attn_fwd_varlen(const void* q, const void* k, const void* v, void* o, float* lse,
                    const int* cu_seqlens, int nseq, int max_seqlen, int total, int Hq, int Hkv,
                    int D, int causal, float scale, hipStream_t stream) {
  int st = check_common(Hq, Hkv, D, causal, scale);
  if (st != ATTN_OK) return st;
  if (nseq < 0 || total < 0 || check_rows(max_seqlen) != ATTN_OK) return ATTN_ERR_SHAPE;
  if ((int64_t)nseq * Hq > (int64_t)1 << 30) return ATTN_ERR_SHAPE;
  if (grid_too_large(nseq, Hq, Hkv, max_seqlen)) return ATTN_ERR_SHAPE;
  if (nseq == 0 || total == 0) return ATTN_OK;
  if (max_seqlen < 1) return ATTN_ERR_VALUE;
  if (!cu_seqlens) return ATTN_ERR_NULL;
  if (reinterpret_cast<uintptr_t>(cu_seqlens) & 3u) return ATTN_ERR_ALIGN;
  return fwd_common(q, k, v, o, lse, packed_layout(cu_seqlens, nseq, max_seqlen, total, Hq, Hkv, D),
                    D, causal, scale, stream);
}

size_t attn_bwd_varlen_workspace_size(int total, int Hq, int Hkv, int D) {
  (void)Hkv;
  (void)D;
  if (total <= 0 || Hq <= 0) return 0;
  return delta_bytes((int64_t)total * Hq);
}

int attn_bwd_varlen_phases(const void* q, const void* k, const void* v, const void* o,
                           const float* lse, const void* dO, void* dq, void* dk, void* dv,
                           const int* cu_seqlens, int nseq, int max_seqlen, int total, int Hq,
                           int Hkv, int D, int causal, float scale, void* workspace,
                           size_t workspace_bytes, int phases, hipStream_t stream) {
  int st = check_common(Hq, Hkv, D, causal, scale);
  if (st != ATTN_OK) return st;
  if (nseq < 0 || total < 0 || check_rows(max_seqlen) != ATTN_OK) return ATTN_ERR_SHAPE;
  if ((int64_t)nseq * Hq > (int64_t)1 << 30) return ATTN_ERR_SHAPE;
  if (grid_too_large(nseq, Hq, Hkv, max_seqlen)) return ATTN_ERR_SHAPE;
  if (!valid_bwd_phases(phases)) return ATTN_ERR_VALUE;
  if (nseq == 0 || total == 0) return ATTN_OK;
  if (max_seqlen < 1) return ATTN_ERR_VALUE;
  if (!cu_seqlens) return ATTN_ERR_NULL;
  if (reinterpret_cast<uintptr_t>(cu_seqlens) & 3u) return ATTN_ERR_ALIGN;
  return bwd_common(q, k, v, o, lse, dO, dq, dk, dv,
                    packed_layout(cu_seqlens, nseq, max_seqlen, total, Hq, Hkv, D), D, causal,
                    scale, workspace, workspace_bytes,
                    attn_bwd_varlen_workspace_size(total, Hq, Hkv, D), phases, stream);
}

int attn_bwd_varlen(const void* q, const void* k, const void* v, const void* o, const float* lse,
                    const void* dO, void* dq, void* dk, void* dv, const int* cu_seqlens, int nseq,
                    int max_seqlen, int total, int Hq, int Hkv, int D, int causal, float scale,
                    void* workspace, size_t workspace_bytes, hipStream_t stream) {
  return attn_bwd_varlen_phases(q, k, v, o, lse, dO, dq, dk, dv, cu_seqlens, nseq, max_seqlen,
                                total, Hq, Hkv, D, causal, scale, workspace, workspace_bytes,
                                ATTN_BWD_DQ | ATTN_BWD_DKDV, stream);
}

size_t attn_fwd_paged_workspace_size(int batch, int max_qlen, int total_q, int max_kvlen,
                                     int Hq, int Hkv, int D) {
  (void)Hkv;
  if (batch <= 0 || max_qlen <= 0 || total_q <= 0 || max_kvlen <= 0 || Hq <= 0 || D <= 0)
    return 0;
  const int split = paged_split(batch, max_qlen, max_kvlen, Hq);
  if (split == 0) return 0;
  const int64_t slots = (int64_t)total_q * Hq * ((max_kvlen + split - 1) / split);
  return round256(slots * D * 4) + round256(slots * 4);
}

int attn_fwd_paged_form(int batch, int max_qlen, int max_kvlen, int Hq, int with_workspace) {
  if (batch < 1 || max_qlen < 1 || max_kvlen < 0 || Hq < 1) return ATTN_ERR_SHAPE;
  if ((int64_t)batch * Hq > (int64_t)1 << 30) return ATTN_ERR_SHAPE;
  if (with_workspace != 0 && with_workspace != 1) return ATTN_ERR_VALUE;
  if (with_workspace && paged_split(batch, max_qlen, max_kvlen, Hq) > 0)
    return ATTN_FWD_PAGED_SPLIT;
  return attn::paged_key_halves((int64_t)batch * Hq, max_qlen) ? ATTN_FWD_PAGED_KEY_HALVES
                                                                : ATTN_FWD_PAGED_UNSPLIT;
}

int attn_fwd_paged(const void* q, const void* k_cache, const void* v_cache, void* o, float* lse,
                   const int* qo_indptr, const int* kv_indptr, const int* kv_indices, int batch,
                   int max_qlen, int total_q, int max_kvlen, int nnz, int num_pages, int Hq,
                   int Hkv, int D, int causal, float scale, void* workspace,
                   size_t workspace_bytes, hipStream_t stream) {
  int st = check_common(Hq, Hkv, D, causal, scale);
  if (st != ATTN_OK) return st;
  if (batch < 0 || total_q < 0 || check_rows(max_qlen) != ATTN_OK) return ATTN_ERR_SHAPE;
  if (check_rows(max_kvlen) != ATTN_OK) return ATTN_ERR_SHAPE;
  if ((st = check_cache(num_pages, nnz, Hkv, D)) != ATTN_OK) return st;
  if ((int64_t)batch * Hq > (int64_t)1 << 30) return ATTN_ERR_SHAPE;
  if (batch == 0 || total_q == 0) return ATTN_OK;
  if (max_qlen < 1) return ATTN_ERR_VALUE;
  if (!qo_indptr || !kv_indptr || (nnz > 0 && !kv_indices)) return ATTN_ERR_NULL;
  if (misaligned4(qo_indptr) || misaligned4(kv_indptr) || misaligned4(kv_indices))
    return ATTN_ERR_ALIGN;
  if (any_null({q, k_cache, v_cache, o, lse})) return ATTN_ERR_NULL;
  if (any_misaligned({q, k_cache, v_cache, o, lse})) return ATTN_ERR_ALIGN;
  Layout L = packed_layout(qo_indptr, batch, max_qlen, total_q, Hq, Hkv, D);
  // The cache [num_pages, Hkv, D] has the packed key layout with a page per row.
  L.kv_cu = kv_indptr;
  L.kv_idx = kv_indices;
  L.nnz = nnz;
  L.num_pages = num_pages;
  // Without a workspace the forward runs unsplit.
  int split = workspace ? paged_split(batch, max_qlen, max_kvlen, Hq) : 0;
  PagedSplit ps{max_kvlen, split, 0, nullptr, nullptr};
  if (split > 0) {
    const size_t need = attn_fwd_paged_workspace_size(batch, max_qlen, total_q, max_kvlen, Hq,
                                                      Hkv, D);
    if (workspace_bytes < need) return ATTN_ERR_WORKSPACE;
    if (misaligned(workspace)) return ATTN_ERR_ALIGN;
    ps.nsplit = (max_kvlen + split - 1) / split;
    const int64_t slots = (int64_t)total_q * Hq * ps.nsplit;
    ps.part_o = static_cast<float*>(workspace);
    ps.part_lse = reinterpret_cast<float*>(static_cast<char*>(workspace) + round256(slots * D * 4));
  }
  return fwd_common(q, k_cache, v_cache, o, lse, L, D, causal, scale, stream, &ps);
}

size_t attn_decode_paged_workspace_size(int batch, int max_kvlen, int Hq, int Hkv, int D) {
  (void)Hkv;
  if (batch <= 0 || max_kvlen <= 0 || Hq <= 0 || D <= 0) return 0;
  const int64_t slots = (int64_t)batch * Hq * decode_chunks(max_kvlen);
  return round256(slots * D * 4) + round256(slots * 4);
}

int attn_decode_paged_phases(const void* q, const void* k_cache, const void* v_cache, void* o,
                             float* lse, const int* kv_indptr, const int* kv_indices, int batch,
                             int max_kvlen, int nnz, int num_pages, int Hq, int Hkv, int D,
                             float scale, void* workspace, size_t workspace_bytes, int phases,
                             hipStream_t stream) {
  int st = check_common(Hq, Hkv, D, 0, scale);
  if (st != ATTN_OK) return st;
  if (phases < 1 || phases > 3) return ATTN_ERR_VALUE;
  if (Hq / Hkv > 32) return ATTN_ERR_GQA;
  if (batch < 0 || check_rows(max_kvlen) != ATTN_OK) return ATTN_ERR_SHAPE;
  if ((st = check_cache(num_pages, nnz, Hkv, D)) != ATTN_OK) return st;
  if ((int64_t)batch * Hq > (int64_t)1 << 30) return ATTN_ERR_SHAPE;
  if (batch == 0) return ATTN_OK;
  if (max_kvlen < 1) return ATTN_ERR_VALUE;
  if (any_null({q, k_cache, v_cache, o, lse, kv_indptr}) || (nnz > 0 && !kv_indices))
    return ATTN_ERR_NULL;
  if (any_misaligned({q, k_cache, v_cache, o, lse})) return ATTN_ERR_ALIGN;
  if (misaligned4(kv_indptr) || misaligned4(kv_indices)) return ATTN_ERR_ALIGN;
  const size_t need = attn_decode_paged_workspace_size(batch, max_kvlen, Hq, Hkv, D);
  if (!workspace || workspace_bytes < need) return ATTN_ERR_WORKSPACE;
  if (misaligned(workspace)) return ATTN_ERR_ALIGN;
  attn::DecodeArgs a;
  a.q = static_cast<const uint16_t*>(q);
  a.k = static_cast<const uint16_t*>(k_cache);
  a.v = static_cast<const uint16_t*>(v_cache);
  a.o = static_cast<uint16_t*>(o);
  a.lse = lse;
  a.kv_cu = kv_indptr;
  a.kv_idx = kv_indices;
  a.batch = batch;
  a.Hq = Hq;
  a.Hkv = Hkv;
  a.group = Hq / Hkv;
  a.nnz = nnz;
  a.num_pages = num_pages;
  a.max_kvlen = max_kvlen;
  a.nchunk = (int)decode_chunks(max_kvlen);
  a.scale_log2 = scale * 1.4426950408889634f;
  const int64_t slots = (int64_t)batch * Hq * a.nchunk;
  a.part_o = static_cast<float*>(workspace);
  a.part_lse = reinterpret_cast<float*>(static_cast<char*>(workspace) + round256(slots * D * 4));
  return attn::launch_decode(a, D, phases, stream) == hipSuccess ? ATTN_OK : ATTN_ERR_HIP;
}

int attn_decode_paged(const void* q, const void* k_cache, const void* v_cache, void* o,
                      float* lse, const int* kv_indptr, const int* kv_indices, int batch,
                      int max_kvlen, int nnz, int num_pages, int Hq, int Hkv, int D, float scale,
                      void* workspace, size_t workspace_bytes, hipStream_t stream) {
  return attn_decode_paged_phases(q, k_cache, v_cache, o, lse, kv_indptr, kv_indices, batch,
                                  max_kvlen, nnz, num_pages, Hq, Hkv, D, scale, workspace,
                                  workspace_bytes, ATTN_DECODE_SPLIT | ATTN_DECODE_MERGE, stream);
}

int attn_gemm_bf16_nt(const void* a, const void* b, void* c, int M, int N, int K,
                      hipStream_t stream) {
  if (M < 0 || N < 0 || K < 0) return ATTN_ERR_SHAPE;
  if (K % 8 != 0 || N % 8 != 0) return ATTN_ERR_SHAPE;
  // 256 rows of an operand must fit the 31-bit offsets of the buffer loads,
  // and the grid must fit one dimension.
  if ((int64_t)K * 2 * 256 > 0x7fffffff) return ATTN_ERR_SHAPE;
  const int64_t tiles = ((int64_t)M + 255) / 256 * (((int64_t)N + 255) / 256);
  if (tiles > 0x7fffffff) return ATTN_ERR_SHAPE;
  if (M == 0 || N == 0) return ATTN_OK;
  // With K == 0 the operands are empty (C = 0) and may be null.
  if (!c || (K > 0 && (!a || !b))) return ATTN_ERR_NULL;
  if (any_misaligned({a, b, c})) return ATTN_ERR_ALIGN;
  attn::GemmArgs g;
  g.a = static_cast<const uint16_t*>(a);
  g.b = static_cast<const uint16_t*>(b);
  g.c = static_cast<uint16_t*>(c);
  g.M = M;
  g.N = N;
  g.K = K;
  g.tiles_m = (M + 255) / 256;
  g.tiles_n = (N + 255) / 256;
  g.tile0 = 0;
  int dev = 0, cus = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
    return ATTN_ERR_HIP;
  return attn::launch_gemm(g, cus, stream) == hipSuccess ? ATTN_OK : ATTN_ERR_HIP;
}

const char* attn_status_string(int status) {
  switch (status) {
    case ATTN_OK: return "ok";
    case ATTN_ERR_NULL: return "a required pointer is null";
    case ATTN_ERR_SHAPE: return "a size is negative, a head count is below 1, or a size is too large";
    case ATTN_ERR_GQA:
      return "Hq is not a multiple of Hkv, or (decode) Hq/Hkv is larger than 32";
    case ATTN_ERR_HEAD_DIM: return "head dimension must be 64, 96 or 128";
    case ATTN_ERR_ALIGN: return "a pointer is not 16-byte aligned";
    case ATTN_ERR_WORKSPACE: return "workspace is null or smaller than the size function returns";
    case ATTN_ERR_HIP: return "a kernel launch failed";
    case ATTN_ERR_VALUE:
      return "scale is not finite and > 0, causal is not 0 or 1, max_seqlen < 1, or a bad phase "
             "mask";
    case ATTN_ERR_SCRATCH:
      return "the backward needs more scratch than attn_bwd_noalloc holds "
             "(ATTN_BWD_NOALLOC_SCRATCH_BYTES)";
    default: return "unknown status";
  }
}

}  // extern "C"
