// Paged decode for gfx950: one new query token per request, attending to the
// request's keys and values in a cache of one token per page (the paged
// decode workload of PTXBench, Appendix A, "Generalization attention
// workloads": grouped-query heads, page size 1, bf16 output and fp32
// log-sum-exp).
//
// Decode reads every key and value once and does little arithmetic with
// them (2 Hq/Hkv FLOP per byte), so it is bound by HBM bandwidth, and a
// request's keys are spread over many workgroups to keep the chip's memory
// system busy:
//
//  * decode_split_kernel: one wavefront per (request, key/value head, chunk
//    of 64 keys).  The query heads of the group are the columns of one MFMA
//    tile.  The chunk's K rows are gathered straight into registers as the A
//    operand of S^T = K Q^T, its V rows into LDS (buffer_load ... lds, one
//    page number per copied row) for the transposing reads of V^T in
//    O^T = V^T P^T; with 16 KiB of LDS per wavefront about ten chunks are in
//    flight on every CU, so the page-number loads and the gathers of all
//    chunks overlap.  A request with one chunk writes its result directly;
//    otherwise the chunk's normalised output and log-sum-exp (base 2) go to
//    the workspace.
//  * decode_merge_kernel: one wavefront per (request, query head) combines
//    the chunks: O = sum_c 2^(L_c - M) O_c / sum_c 2^(L_c - M), with M the
//    largest L_c, and L = M + log2 sum_c 2^(L_c - M), returned as a natural
//    log.
#include "attn_kernels.hpp"
#include "device_common.hpp"

namespace attn {
namespace {

static_assert(kDecodeChunk == 64, "one 64-key chunk per wavefront");

template <int D>
__global__ __launch_bounds__(64) void decode_split_kernel(DecodeArgs a) {
  using Tile = AsyncTile<D, 1>;
  constexpr int P = Tile::P;
  __shared__ __attribute__((aligned(1024))) uint16_t sv[Tile::ELEMS];   // the chunk's V rows

  const int lane = threadIdx.x, l32 = lane & 31, half = lane >> 5;
  const int z = blockIdx.x / a.Hkv, hk = blockIdx.x % a.Hkv;
  const int chunk = blockIdx.y;
  const int G = a.group;

  int ks = a.kv_cu[z], ke = a.kv_cu[z + 1];
  ks = ks < 0 ? 0 : (ks > a.nnz ? a.nnz : ks);
  ke = ke < ks ? ks : (ke > a.nnz ? a.nnz : ke);
  const int len = min(ke - ks, a.max_kvlen);
  const int k0 = chunk * kDecodeChunk;
  if (k0 >= len) return;
  const int nch = (len + kDecodeChunk - 1) / kDecodeChunk;

  // Lane i fetches the page of key k0 + i; other lanes' pages come by
  // cross-lane reads.  Keys past the end and pages outside the cache read
  // as zero rows.
  const rsrc_t ixr = make_rsrc(a.kv_idx + ks, (int64_t)len * 4);
  const int page = bload4(ixr, 4 * (k0 + lane));
  const bool ok = k0 + lane < len && (unsigned)page < (unsigned)a.num_pages;
  const int row_bytes = a.Hkv * D * 2;
  const int my_off = ok ? page * row_bytes : kPadOffset;

  // Q^T as the B operand: column l32 is query head hk * G + l32 of the
  // request; columns >= G read as zero.
  const int64_t qoff = ((int64_t)z * a.Hq + (int64_t)hk * G) * D;
  const rsrc_t rq = make_rsrc(a.q + qoff, (int64_t)G * D * 2);
  u32x4 qreg[D / 16];
#pragma unroll
  for (int c = 0; c < D / 16; ++c) qreg[c] = bload16(rq, l32 * D * 2 + 16 * half + 32 * c);

  const int64_t cache_bytes = (int64_t)a.num_pages * row_bytes - (int64_t)hk * D * 2;
  const rsrc_t kc = make_rsrc(a.k + (int64_t)hk * D, cache_bytes);
  const rsrc_t vc = make_rsrc(a.v + (int64_t)hk * D, cache_bytes);

  // V rows gathered into LDS (DMA instruction j copies tile rows 4j + lane/16
  // at D = 128), K rows straight into registers as the A operand of
  // S^T = K Q^T: block b holds keys 32b + l32, 16 bytes at column 16c + 8 half.
  {
    const Tile dma(0, lane, 0);
    int off[Tile::NJ];
#pragma unroll
    for (int j = 0; j < Tile::NJ; ++j) {
      const int c = Tile::chunk_of(0, j, lane);
      const int ro = __shfl(my_off, Tile::row_of(0, j, lane));
      off[j] = c < D / 8 ? ro + 16 * c : kPadOffset;
    }
    dma.load_at(vc, off, sv, 0);
  }
  u32x4 kreg[2][D / 16];
#pragma unroll
  for (int b = 0; b < 2; ++b) {
    const int ro = __shfl(my_off, 32 * b + l32);
#pragma unroll
    for (int c = 0; c < D / 16; ++c) kreg[b][c] = bload16(kc, ro + 16 * half + 32 * c);
  }

  f32x16 s[2];
#pragma unroll
  for (int b = 0; b < 2; ++b) {
#pragma unroll
    for (int r = 0; r < 16; ++r) s[b][r] = 0.f;
#pragma unroll
    for (int c = 0; c < D / 16; ++c) s[b] = mfma32(kreg[b][c], qreg[c], s[b]);
  }
  // s[b][r]: key k0 + 32b + 8(r/4) + 4half + r%4, query column l32.
  float mx = -INFINITY;
#pragma unroll
  for (int b = 0; b < 2; ++b)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int key = k0 + 32 * b + 8 * (r / 4) + 4 * half + (r % 4);
      s[b][r] = key < len ? s[b][r] : -INFINITY;
      mx = fmaxf(mx, s[b][r]);
    }
  mx = max_halves(mx);
  const float mt = mx * a.scale_log2;   // the chunk's row maximum, exp2 units (finite)
  float ls = 0.f;
#pragma unroll
  for (int b = 0; b < 2; ++b)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      s[b][r] = fast_exp2(__builtin_fmaf(s[b][r], a.scale_log2, -mt));
      ls += s[b][r];
    }
  ls = sum_halves(ls);

  // O^T[d][q] = sum over the chunk's keys of V^T[d][key] P^T[key][q], V^T
  // read transposed out of the V tile (chunk c of block b = tile rows
  // 32b + 16c .. + 15).
  wait_vm<0>();   // the V rows have landed (one wavefront: no barrier needed)
  const TransReader<D> tr(lane);
  f32x16 oacc[D / 32];
#pragma unroll
  for (int db = 0; db < D / 32; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) oacc[db][r] = 0.f;
#pragma unroll
  for (int b = 0; b < 2; ++b)
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      const u32x4 pb = pack_chunk(s[b], c);
      const int rc = 16 * (2 * b + c) * P;
#pragma unroll
      for (int db = 0; db < D / 32; ++db) {
        const u32x2 lo = ld_tr(sv + tr.tr[db][0] + rc), hi = ld_tr(sv + tr.tr[db][1] + rc);
        oacc[db] = mfma32(u32x4{lo[0], lo[1], hi[0], hi[1]}, pb, oacc[db]);
      }
    }

  // Lane (l32, half) holds column l32 (query head hk G + l32) at rows
  // 32 db + 8 i + 4 half + 0..3.
  if (l32 >= G) return;
  const float inv = 1.f / ls;   // ls >= 1: the maximum's own key contributes 1
  const float lse2 = mt + log2f(ls);
  const int64_t h = (int64_t)hk * G + l32;
  if (nch == 1) {
    uint16_t* op = a.o + ((int64_t)z * a.Hq + h) * D + 4 * half;
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
      for (int i = 0; i < 4; ++i)
        st8(op + 32 * db + 8 * i,
            u32x2{pack_bf16(oacc[db][4 * i] * inv, oacc[db][4 * i + 1] * inv),
                  pack_bf16(oacc[db][4 * i + 2] * inv, oacc[db][4 * i + 3] * inv)});
    if (half == 0) a.lse[h * a.batch + z] = lse2 * kLn2;
  } else {
    const int64_t slot = ((int64_t)z * a.Hq + h) * a.nchunk + chunk;
    float* po = a.part_o + slot * D + 4 * half;
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
      for (int i = 0; i < 4; ++i)
        *reinterpret_cast<f32x4*>(po + 32 * db + 8 * i) =
            f32x4{oacc[db][4 * i], oacc[db][4 * i + 1], oacc[db][4 * i + 2], oacc[db][4 * i + 3]} *
            inv;
    if (half == 0) a.part_lse[slot] = lse2;
  }
}

// One wavefront per (request, query head).  Lane group gq = lane / CW takes
// chunks gq, gq + NG, ... and lane l % CW output columns 4 (l % CW) .. + 3
// (lanes past column D idle); the groups' sums are added with cross-lane
// exchanges.  The first BATCH chunks' partial outputs and the first 64
// log-sum-exps (one per lane) are loaded before the request's length is
// known: they lie inside the workspace rows of this (request, head), and the
// slots past the request's chunks, which hold stale values, are discarded by
// selects.  So a request of up to BATCH chunks costs one memory round trip.
template <int D>
__global__ __launch_bounds__(64) void decode_merge_kernel(DecodeArgs a) {
  constexpr int CW = D / 4 <= 16 ? 16 : 32;   // lanes per output row (a power of two)
  constexpr int NG = 64 / CW;                 // lane groups
  constexpr int U = 16;                       // chunks per lane group and batch
  constexpr int BATCH = NG * U;               // 32 or 64 chunks
  static_assert(BATCH <= 64, "first-batch weights come from one lane each");
  const int lane = threadIdx.x;
  const int z = blockIdx.x / a.Hq, h = blockIdx.x % a.Hq;
  const int gq = lane / CW, d = 4 * (lane % CW);
  const bool col = d < D;
  const int nck = a.nchunk;
  const int64_t slot0 = ((int64_t)z * a.Hq + h) * nck;
  const float* const po = a.part_o + slot0 * D + d;
  const float* const pl = a.part_lse + slot0;

  // Range-checked loads (zero past this (request, head)'s slots or past
  // column D), with no branch between them.
  const rsrc_t ro = make_rsrc(a.part_o + slot0 * D, (int64_t)nck * D * 4);
  const rsrc_t rl = make_rsrc(pl, (int64_t)nck * 4);
  const int dcol = col ? 4 * d : kPadOffset;
  f32x4 v[U];
#pragma unroll
  for (int u = 0; u < U; ++u)
    v[u] = __builtin_bit_cast(f32x4, bload16(ro, dcol + 4 * D * (gq + NG * u)));
  const float l0 = lane < nck ? __int_as_float(bload4(rl, 4 * lane)) : -INFINITY;

  int ks = a.kv_cu[z], ke = a.kv_cu[z + 1];
  ks = ks < 0 ? 0 : (ks > a.nnz ? a.nnz : ks);
  ke = ke < ks ? ks : (ke > a.nnz ? a.nnz : ke);
  const int len = min(ke - ks, a.max_kvlen);
  const int nch = (len + kDecodeChunk - 1) / kDecodeChunk;
  if (nch == 1) return;   // written by the split kernel
  uint16_t* op = a.o + ((int64_t)z * a.Hq + h) * D + d;
  if (nch == 0) {   // no keys: O = 0, L = -inf
    if (gq == 0 && col) st8(op, u32x2{0u, 0u});
    if (lane == 0) a.lse[(int64_t)h * a.batch + z] = -INFINITY;
    return;
  }

  // M = max over the request's chunks of L_c, then the weights 2^(L_c - M)
  // (lane c holds chunk c's weight for the first 64 chunks).
  float M = lane < nch ? l0 : -INFINITY;
  for (int c0 = 64; c0 < nch; c0 += 64)
    if (c0 + lane < nch) M = fmaxf(M, pl[c0 + lane]);
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) M = fmaxf(M, __shfl_xor(M, o));
  const float wl = lane < nch ? fast_exp2(l0 - M) : 0.f;
  float wsum = wl;
  for (int c0 = 64; c0 < nch; c0 += 64)
    if (c0 + lane < nch) wsum += fast_exp2(pl[c0 + lane] - M);

  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int u = 0; u < U; ++u) {
    const int c = gq + NG * u;
    const float w = __shfl(wl, c);
    if (c < nch) acc += w * v[u];
  }
  for (int cb = BATCH; cb < nch; cb += BATCH) {
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int c = cb + gq + NG * u;
      if (c < nch && col)
        acc += fast_exp2(pl[c] - M) * *reinterpret_cast<const f32x4*>(po + (int64_t)c * D);
    }
  }
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) wsum += __shfl_xor(wsum, o);
#pragma unroll
  for (int o = CW; o < 64; o <<= 1)
#pragma unroll
    for (int i = 0; i < 4; ++i) acc[i] += __shfl_xor(acc[i], o);
  const float inv = 1.f / wsum;
  if (gq == 0 && col)
    st8(op, u32x2{pack_bf16(acc[0] * inv, acc[1] * inv), pack_bf16(acc[2] * inv, acc[3] * inv)});
  if (lane == 0) a.lse[(int64_t)h * a.batch + z] = (M + log2f(wsum)) * kLn2;
}

template __global__ void decode_split_kernel<64>(DecodeArgs);
template __global__ void decode_split_kernel<96>(DecodeArgs);
template __global__ void decode_split_kernel<128>(DecodeArgs);
template __global__ void decode_merge_kernel<64>(DecodeArgs);
template __global__ void decode_merge_kernel<96>(DecodeArgs);
template __global__ void decode_merge_kernel<128>(DecodeArgs);

template <int D>
void launch_decode_d(const DecodeArgs& a, int phases, hipStream_t stream) {
  if (phases & 1) {
    const dim3 gs((unsigned)(a.batch * a.Hkv), (unsigned)a.nchunk);
    hipLaunchKernelGGL((decode_split_kernel<D>), gs, dim3(64), 0, stream, a);
  }
  if (phases & 2)
    hipLaunchKernelGGL((decode_merge_kernel<D>), dim3((unsigned)(a.batch * a.Hq)), dim3(64), 0,
                       stream, a);
}

}  // namespace

hipError_t launch_decode(const DecodeArgs& a, int D, int phases, hipStream_t stream) {
  if (D == 64)
    launch_decode_d<64>(a, phases, stream);
  else if (D == 96)
    launch_decode_d<96>(a, phases, stream);
  else
    launch_decode_d<128>(a, phases, stream);
  return hipGetLastError();
}

}  // namespace attn
