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
//  * decode_split_kernel: one workgroup of 4 wavefronts per (request,
//    key/value head, chunk of 128 keys).  The rows of the chunk are gathered
//    from the cache straight into LDS (buffer_load ... lds, one page number per
//    copied row).  The query heads of the group are the columns of one MFMA
//    tile: each wavefront computes S^T = K Q^T for 32 keys, the workgroup
//    agrees on one maximum per query through LDS, and each wavefront adds
//    P^T into O^T = V^T P^T with V^T read transposed out of the V tile.  The
//    four partial outputs share that maximum, so they are summed without
//    rescaling.  A request with one chunk writes its result directly;
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

constexpr int kWaves = 4;
constexpr int kThreads = 64 * kWaves;
static_assert(kDecodeChunk == 32 * kWaves, "one 32-key block per wavefront");

template <int D>
__global__ __launch_bounds__(kThreads, 2) void decode_split_kernel(DecodeArgs a) {
  using Tile = AsyncTile<D, kWaves>;
  constexpr int P = Tile::P;
  // K tiles (keys 0-63, 64-127) then V tiles; reused for the cross-wavefront
  // sum of O^T once every wavefront has finished reading them.
  __shared__ __attribute__((aligned(1024))) uint16_t smem[4 * Tile::ELEMS];
  __shared__ float red_m[kWaves][32];
  __shared__ float red_l[kWaves][32];

  const int lane = threadIdx.x & 63, wave = wave_id();
  const int l32 = lane & 31, half = lane >> 5;
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

  // Page numbers of this lane's rows in the four tile copies (the same rows
  // for K and V).
  const rsrc_t ixr = make_rsrc(a.kv_idx + ks, (int64_t)len * 4);
  int pidx[2][Tile::NJ];
#pragma unroll
  for (int t = 0; t < 2; ++t)
#pragma unroll
    for (int j = 0; j < Tile::NJ; ++j)
      pidx[t][j] = bload4(ixr, 4 * (k0 + 64 * t + Tile::row_of(wave, j, lane)));

  // Q^T as the B operand: column l32 is query head hk * G + l32 of the
  // request; columns >= G read as zero.
  const int64_t qoff = ((int64_t)z * a.Hq + (int64_t)hk * G) * D;
  const rsrc_t rq = make_rsrc(a.q + qoff, (int64_t)G * D * 2);
  u32x4 qreg[D / 16];
#pragma unroll
  for (int c = 0; c < D / 16; ++c) qreg[c] = bload16(rq, l32 * D * 2 + 16 * half + 32 * c);

  const int row_bytes = a.Hkv * D * 2;
  const int64_t cache_bytes = (int64_t)a.num_pages * row_bytes - (int64_t)hk * D * 2;
  const rsrc_t kc = make_rsrc(a.k + (int64_t)hk * D, cache_bytes);
  const rsrc_t vc = make_rsrc(a.v + (int64_t)hk * D, cache_bytes);
  const Tile dma(wave, lane, 0);
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    int off[Tile::NJ];
#pragma unroll
    for (int j = 0; j < Tile::NJ; ++j) {
      const int key = k0 + 64 * t + Tile::row_of(wave, j, lane);
      off[j] = Tile::gather_off(wave, j, lane, pidx[t][j], key < len, a.num_pages, row_bytes);
    }
    dma.load_at(kc, off, smem + t * Tile::ELEMS, wave);
    dma.load_at(vc, off, smem + (2 + t) * Tile::ELEMS, wave);
  }
  wait_vm<0>();
  __syncthreads();

  // S^T for this wavefront's keys kw0 .. kw0 + 31 (tile wave / 2).
  const int kw0 = k0 + 32 * wave;
  const RowReader<D> rr(l32, half);
  const uint16_t* kt = smem + (wave >> 1) * Tile::ELEMS + 32 * (wave & 1) * P;
  f32x16 s;
#pragma unroll
  for (int r = 0; r < 16; ++r) s[r] = 0.f;
#pragma unroll
  for (int c = 0; c < D / 16; ++c) s = mfma32(ld16(kt + rr.rm[c]), qreg[c], s);
  // s[r]: key kw0 + 8(r/4) + 4half + r%4, query column l32.
  float mx = -INFINITY;
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int key = kw0 + 8 * (r / 4) + 4 * half + (r % 4);
    s[r] = key < len ? s[r] : -INFINITY;
    mx = fmaxf(mx, s[r]);
  }
  mx = fmaxf(mx, swap_halves(mx));
  if (half == 0) red_m[wave][l32] = mx;
  __syncthreads();
  float m = red_m[0][l32];
#pragma unroll
  for (int w = 1; w < kWaves; ++w) m = fmaxf(m, red_m[w][l32]);
  const float mt = m * a.scale_log2;   // the chunk's row maximum, exp2 units (finite)
  float ls = 0.f;
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    s[r] = fast_exp2(__builtin_fmaf(s[r], a.scale_log2, -mt));
    ls += s[r];
  }
  ls += swap_halves(ls);

  // O^T[d][q] += sum over this wavefront's keys of V^T[d][key] P^T[key][q].
  const TransReader<D> tr(lane);
  const uint16_t* vt = smem + (2 + (wave >> 1)) * Tile::ELEMS;
  f32x16 oacc[D / 32];
#pragma unroll
  for (int db = 0; db < D / 32; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) oacc[db][r] = 0.f;
#pragma unroll
  for (int c = 0; c < 2; ++c) {
    const u32x4 pb = pack_chunk(s, c);
    const int rc = 16 * (2 * (wave & 1) + c) * P;
#pragma unroll
    for (int db = 0; db < D / 32; ++db) {
      const u32x2 lo = ld_tr(vt + tr.tr[db][0] + rc), hi = ld_tr(vt + tr.tr[db][1] + rc);
      oacc[db] = mfma32(u32x4{lo[0], lo[1], hi[0], hi[1]}, pb, oacc[db]);
    }
  }

  // Sum over the wavefronts: each writes its G valid columns, [wave][g][D]
  // fp32 (at most 4 x 32 x D x 4 bytes, within the tile buffer).
  __syncthreads();   // every wavefront is done with the tiles
  float* red_o = reinterpret_cast<float*>(smem);
  if (l32 < G) {
    float* dst = red_o + ((int64_t)wave * G + l32) * D;
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
      for (int g = 0; g < 4; ++g)
        *reinterpret_cast<f32x4*>(dst + 32 * db + 8 * g + 4 * half) =
            f32x4{oacc[db][4 * g], oacc[db][4 * g + 1], oacc[db][4 * g + 2], oacc[db][4 * g + 3]};
  }
  if (half == 0) red_l[wave][l32] = ls;
  __syncthreads();

  const int64_t hq0 = (int64_t)hk * G;
  for (int i = threadIdx.x; i < G * (D / 4); i += kThreads) {
    const int g = i / (D / 4), d = 4 * (i % (D / 4));
    f32x4 acc = *reinterpret_cast<const f32x4*>(red_o + (int64_t)g * D + d);
    float l = red_l[0][g], mg = red_m[0][g];
#pragma unroll
    for (int w = 1; w < kWaves; ++w) {
      const f32x4 x = *reinterpret_cast<const f32x4*>(red_o + ((int64_t)w * G + g) * D + d);
      acc += x;
      l += red_l[w][g];
      mg = fmaxf(mg, red_m[w][g]);
    }
    const float inv = 1.f / l;   // l >= 1: the maximum's own key contributes 1
    const float lse2 = mg * a.scale_log2 + log2f(l);
    const int64_t h = hq0 + g;
    if (nch == 1) {
      uint16_t* op = a.o + ((int64_t)z * a.Hq + h) * D + d;
      st8(op, u32x2{pack_bf16(acc[0] * inv, acc[1] * inv), pack_bf16(acc[2] * inv, acc[3] * inv)});
      if (d == 0) a.lse[h * a.batch + z] = lse2 * kLn2;
    } else {
      const int64_t slot = ((int64_t)z * a.Hq + h) * a.nchunk + chunk;
      *reinterpret_cast<f32x4*>(a.part_o + slot * D + d) = acc * inv;
      if (d == 0) a.part_lse[slot] = lse2;
    }
  }
}

// One wavefront per (request, query head); lane l handles output columns
// 4l .. 4l + 3.
template <int D>
__global__ __launch_bounds__(64) void decode_merge_kernel(DecodeArgs a) {
  const int lane = threadIdx.x;
  const int z = blockIdx.x / a.Hq, h = blockIdx.x % a.Hq;
  int ks = a.kv_cu[z], ke = a.kv_cu[z + 1];
  ks = ks < 0 ? 0 : (ks > a.nnz ? a.nnz : ks);
  ke = ke < ks ? ks : (ke > a.nnz ? a.nnz : ke);
  const int len = min(ke - ks, a.max_kvlen);
  const int nch = (len + kDecodeChunk - 1) / kDecodeChunk;
  if (nch == 1) return;   // written by the split kernel
  const int d = 4 * lane;
  uint16_t* op = a.o + ((int64_t)z * a.Hq + h) * D + d;
  if (nch == 0) {   // no keys: O = 0, L = -inf
    if (d < D) st8(op, u32x2{0u, 0u});
    if (lane == 0) a.lse[(int64_t)h * a.batch + z] = -INFINITY;
    return;
  }
  const int64_t slot0 = ((int64_t)z * a.Hq + h) * a.nchunk;
  float M = -INFINITY;
  for (int c = 0; c < nch; ++c) M = fmaxf(M, a.part_lse[slot0 + c]);
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  float wsum = 0.f;
  for (int c = 0; c < nch; ++c) {
    const float w = fast_exp2(a.part_lse[slot0 + c] - M);
    wsum += w;
    if (d < D) acc += w * *reinterpret_cast<const f32x4*>(a.part_o + (slot0 + c) * D + d);
  }
  const float inv = 1.f / wsum;
  if (d < D)
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
void launch_decode_d(const DecodeArgs& a, hipStream_t stream) {
  const dim3 gs((unsigned)(a.batch * a.Hkv), (unsigned)a.nchunk);
  hipLaunchKernelGGL((decode_split_kernel<D>), gs, dim3(kThreads), 0, stream, a);
  hipLaunchKernelGGL((decode_merge_kernel<D>), dim3((unsigned)(a.batch * a.Hq)), dim3(64), 0,
                     stream, a);
}

}  // namespace

hipError_t launch_decode(const DecodeArgs& a, int D, hipStream_t stream) {
  if (D == 64)
    launch_decode_d<64>(a, stream);
  else if (D == 96)
    launch_decode_d<96>(a, stream);
  else
    launch_decode_d<128>(a, stream);
  return hipGetLastError();
}

}  // namespace attn
