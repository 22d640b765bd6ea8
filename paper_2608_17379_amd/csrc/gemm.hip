// BF16 GEMM C = A B^T for gfx950 (the fifth primary workload of PTXBench,
// Appendix A, "Workloads": A [M, K], B [N, K], C [M, N], all bf16, both
// operands with the reduction index contiguous), fp32 accumulation on MFMA.
//
// One workgroup of 8 wavefronts per 256 x 256 tile of C, one workgroup per
// CU.  Each K step of 64 copies the A and B tiles (256 rows x 128 bytes
// each) straight from global memory into a two-stage LDS ring
// (buffer_load ... lds, issued a step ahead and spread over the step's K
// chunks), in the swizzled row-major
// layout of the attention kernels, so that every MFMA operand is one
// conflict-free 16-byte LDS read.  Wavefront (wm, wn) owns rows
// 128 wm .. + 127 of the tile and columns 64 wn .. + 63, as 4 x 2 blocks of
// 32 x 32, and computes them transposed (C^T block = B rows x A rows), so
// that each lane holds four consecutive columns of one row of C and stores
// them as 8 bytes.
//
// With one workgroup per CU the tiles run in rounds of one per CU; when the
// last round would be at most half full, its tiles are computed as 128-row
// halves (8 wavefronts of 64 x 64 each), which fills the chip for half a
// round instead of half the chip for a whole one.  Such a call is one launch
// of one workgroup per CU that runs its full tiles and then its half tile
// (gemm_rounds_kernel); any other runs one workgroup per tile.
//
// Tiles are assigned XCD by XCD: the hardware hands workgroup ids to the 8
// XCDs in turn, so workgroup b runs on XCD b % 8; the tiles are numbered so
// that each XCD receives a contiguous range, walked in bands of 4 row tiles
// (all column tiles of the band, four rows at a time), which keeps the A and
// B slabs of the tiles running together on one XCD in its L2.
//
// Rows past M or N read as zero through buffer-range checks and are not
// stored; a K that is not a multiple of 64 reads zeros past K (K is a
// multiple of 8, so every 16-byte chunk is wholly inside or outside).
#include "attn_kernels.hpp"
#include "device_common.hpp"

namespace attn {
namespace {

constexpr int kTM = 256, kTN = 256, kTK = 64;
constexpr int kWaves = 8;
constexpr int kThreads = 64 * kWaves;
constexpr int kBand = 4;   // row tiles per band of the tile order

using GTile = AsyncTile<64, kWaves>;   // one [64 rows][64 k] sub-tile per DMA instruction
static_assert(GTile::NJ == 1, "one DMA instruction per wavefront per 64-row sub-tile");
static_assert(kTK / 16 == 4, "one 64-row sub-tile copied per 16-wide K chunk");
constexpr int kSubElems = GTile::ELEMS;            // 4096 bf16
constexpr int kTileElems = 4 * kSubElems;          // 256 rows

// Tile t of the tile order (TM = 256), or its 128-row half hm (TM = 128),
// by the whole workgroup, on the LDS stages (sa0, sb0) and (sa1, sb1).
template <int TM, bool KTAIL>
__device__ __forceinline__ void gemm_tile(const GemmArgs& g, int t, int hm, uint16_t* sa0,
                                          uint16_t* sb0, uint16_t* sa1, uint16_t* sb1) {
  constexpr int ASUB = TM / 64;   // 64-row sub-tiles of the A tile
  constexpr int MB = TM / 64;     // 32-row blocks of each wavefront (4 or 2)
  constexpr int NB = 2;           // 32-column blocks of each wavefront

  const int lane = threadIdx.x & 63, wave = wave_id();
  const int l32 = lane & 31, half = lane >> 5;

  const int band_tiles = kBand * g.tiles_n;
  const int m_first = (t / band_tiles) * kBand;
  const int band_rows = min(kBand, g.tiles_m - m_first);
  const int tb = t % band_tiles;
  const int m0 = (m_first + tb % band_rows) * kTM + hm * TM;
  const int n0 = (tb / band_rows) * kTN;

  const int K = g.K;
  const int row_bytes = K * 2;
  const rsrc_t ra = make_rsrc(g.a + (int64_t)m0 * K, (int64_t)(g.M - m0) * row_bytes);
  const rsrc_t rb = make_rsrc(g.b + (int64_t)n0 * K, (int64_t)(g.N - n0) * row_bytes);

  // This lane's DMA source: row r = 8 wave + lane / 8 of every 64-row
  // sub-tile, logical 16-byte chunk lg (k = 8 lg .. 8 lg + 7 of the step).
  const int drow = GTile::row_of(wave, 0, lane);
  const int lg = GTile::chunk_of(wave, 0, lane);
  const int doff = drow * row_bytes + 16 * lg;

  // Copies of 64-row sub-tile s of step kt (A, when the tile has it, and B).
  auto load_part = [&](int kt, int s, uint16_t* da, uint16_t* db) __attribute__((always_inline)) {
    const int k0 = kt * kTK;
    int off = doff + 64 * s * row_bytes + 2 * k0;
    if constexpr (KTAIL) off = k0 + 8 * lg < K ? off : kPadOffset;
    if (s < ASUB)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          ra, (ATTN_LDS void*)(da + s * kSubElems + wave * 64 * 8), 16, off, 0, 0, 0);
    __builtin_amdgcn_raw_ptr_buffer_load_lds(
        rb, (ATTN_LDS void*)(db + s * kSubElems + wave * 64 * 8), 16, off, 0, 0, 0);
  };

  const int wm = wave >> 2, wn = wave & 3;   // rows (TM / 2) wm .., columns 64 wn ..
  const RowReader<64> rr(l32, half);
  // 32-row block q of a 256-row tile starts at element q * 2048 (sub-tile
  // q / 2, row 32 (q % 2)); the swizzle depends on the row modulo 16 only.
  f32x16 acc[NB][MB];
#pragma unroll
  for (int j = 0; j < NB; ++j)
#pragma unroll
    for (int i = 0; i < MB; ++i)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[j][i][r] = 0.f;

  // One step's products on stage (sa, sb).  When `next` is set, the copies
  // of step kt_next into (na, nb) are spread over the step, one sub-tile per
  // 16-wide K chunk, instead of leaving in one burst.
  auto compute = [&](const uint16_t* sa, const uint16_t* sb, bool next, int kt_next, uint16_t* na,
                     uint16_t* nb) __attribute__((always_inline)) {
#pragma unroll
    for (int c = 0; c < kTK / 16; ++c) {
      u32x4 bo[NB], ao[MB];
#pragma unroll
      for (int j = 0; j < NB; ++j) bo[j] = ld16(sb + (NB * wn + j) * 2048 + rr.rm[c]);
#pragma unroll
      for (int i = 0; i < MB; ++i) ao[i] = ld16(sa + (MB * wm + i) * 2048 + rr.rm[c]);
      // The copies go out at raised wave priority, ahead of the other
      // wavefront's MFMA and LDS issue on the SIMD, so that they have as much
      // of the step as possible to land.
      if (next) {
        __builtin_amdgcn_s_setprio(3);
        load_part(kt_next, c, na, nb);
        __builtin_amdgcn_s_setprio(0);
      }
#pragma unroll
      for (int j = 0; j < NB; ++j)
#pragma unroll
        for (int i = 0; i < MB; ++i) acc[j][i] = mfma32(bo[j], ao[i], acc[j][i]);
    }
  };

  const int nkt = (K + kTK - 1) / kTK;
  // Step kt: wait for its copies (this wavefront's, then everyone's through
  // the barrier, which also frees the stage read at kt - 1), then compute,
  // copying kt + 1 into that stage along the way.
  auto step = [&](int kt, const uint16_t* ca, const uint16_t* cb, uint16_t* na, uint16_t* nb)
      __attribute__((always_inline)) {
    wait_vm<0>();
    __syncthreads();
    compute(ca, cb, kt + 1 < nkt, kt + 1, na, nb);
  };
  if (nkt > 0) {
#pragma unroll
    for (int s = 0; s < 4; ++s) load_part(0, s, sa0, sb0);
  }
  int kt = 0;
  for (; kt + 1 < nkt; kt += 2) {
    step(kt, sa0, sb0, sa1, sb1);
    step(kt + 1, sa1, sb1, sa0, sb0);
  }
  if (kt < nkt) step(kt, sa0, sb0, sa1, sb1);

  // acc[j][i] is the C^T block of columns n0 + 64 wn + 32 j + (8 (r/4) +
  // 4 half + r%4) and row m0 + (TM / 2) wm + 32 i + l32.
#pragma unroll
  for (int i = 0; i < MB; ++i) {
    const int m = m0 + (TM / 2) * wm + 32 * i + l32;
    if (m >= g.M) continue;
    uint16_t* crow = g.c + (int64_t)m * g.N;
#pragma unroll
    for (int j = 0; j < NB; ++j)
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int n = n0 + 64 * wn + 32 * j + 8 * q + 4 * half;
        if (n < g.N)
          st8(crow + n, u32x2{pack_bf16(acc[j][i][4 * q], acc[j][i][4 * q + 1]),
                              pack_bf16(acc[j][i][4 * q + 2], acc[j][i][4 * q + 3])});
      }
  }
}

// TM = 256: workgroup b computes tile g.tile0 + b (in the order below).
// TM = 128: workgroups 2 i and 2 i + 1 compute the two 128-row halves of
// tile g.tile0 + i.
template <int TM, bool KTAIL>
__global__ __launch_bounds__(kThreads, 1) void gemm_nt_kernel(GemmArgs g) {
  constexpr int ASUB = TM / 64;
  __shared__ __attribute__((aligned(1024))) uint16_t sa0[ASUB * kSubElems];
  __shared__ __attribute__((aligned(1024))) uint16_t sb0[kTileElems];
  __shared__ __attribute__((aligned(1024))) uint16_t sa1[ASUB * kSubElems];
  __shared__ __attribute__((aligned(1024))) uint16_t sb1[kTileElems];
  const int nblk = (int)gridDim.x, bid = (int)blockIdx.x;
  const int w = nblk % 8 == 0 ? (bid % 8) * (nblk / 8) + bid / 8 : bid;
  gemm_tile<TM, KTAIL>(g, g.tile0 + (TM == kTM ? w : w / 2), TM == kTM ? 0 : w % 2, sa0, sb0,
                       sa1, sb1);
}

// The whole call in one launch of one workgroup per CU (gridDim.x, a
// multiple of 8 that divides full): the first full tiles in rounds, each
// workgroup taking the tiles that workgroups bid, bid + gridDim.x, ... of
// gemm_nt_kernel<256> would take (so the XCD of every tile is the same),
// then the 128-row halves of the remaining tiles, as the workgroups of
// gemm_nt_kernel<128> would take them.  Each workgroup thus runs its last
// round's half tile right after its full tiles, with no second launch.
struct RoundsArgs {
  GemmArgs g;
  int full;   // tiles run whole, in rounds (a multiple of gridDim.x)
};

template <bool KTAIL>
__global__ __launch_bounds__(kThreads, 1) void gemm_rounds_kernel(RoundsArgs args) {
  const GemmArgs& g = args.g;
  __shared__ __attribute__((aligned(1024))) uint16_t sa0[kTileElems];
  __shared__ __attribute__((aligned(1024))) uint16_t sb0[kTileElems];
  __shared__ __attribute__((aligned(1024))) uint16_t sa1[kTileElems];
  __shared__ __attribute__((aligned(1024))) uint16_t sb1[kTileElems];
  const int nblk = (int)gridDim.x, bid = (int)blockIdx.x;
  const int x = bid % 8, j = bid / 8, per = nblk / 8;
  const int full = args.full;
  const int rounds = full / nblk;
  for (int r = 0; r < rounds; ++r) {
    gemm_tile<kTM, KTAIL>(g, x * (full / 8) + j + per * r, 0, sa0, sb0, sa1, sb1);
    __syncthreads();   // every wavefront is done with the stages
  }
  const int nhalf = 2 * (g.tiles_m * g.tiles_n - full);
  if (bid < nhalf) {
    const int w = nhalf % 8 == 0 ? x * (nhalf / 8) + j : bid;
    gemm_tile<128, KTAIL>(g, full + w / 2, w % 2, sa0, sb0, sa1, sb1);
  }
}

template __global__ void gemm_rounds_kernel<false>(RoundsArgs);
template __global__ void gemm_rounds_kernel<true>(RoundsArgs);
template __global__ void gemm_nt_kernel<256, false>(GemmArgs);
template __global__ void gemm_nt_kernel<256, true>(GemmArgs);
template __global__ void gemm_nt_kernel<128, false>(GemmArgs);
template __global__ void gemm_nt_kernel<128, true>(GemmArgs);

template <int TM>
void launch_part(const GemmArgs& g, int nwg, hipStream_t stream) {
  if (nwg <= 0) return;
  if (g.K % kTK != 0)
    hipLaunchKernelGGL((gemm_nt_kernel<TM, true>), dim3((unsigned)nwg), dim3(kThreads), 0,
                       stream, g);
  else
    hipLaunchKernelGGL((gemm_nt_kernel<TM, false>), dim3((unsigned)nwg), dim3(kThreads), 0,
                       stream, g);
}

}  // namespace

// One workgroup per CU runs at a time, so the tiles go in rounds of `cus`.
// When the last round would be at most half full, its tiles are split into
// 128-row halves in a second launch: twice as many workgroups, each half as
// long, so the last round takes half the time of a full one.
hipError_t launch_gemm(const GemmArgs& g, int cus, hipStream_t stream) {
  const int tiles = g.tiles_m * g.tiles_n;
  const int rem = cus > 0 ? tiles % cus : 0;
  const bool split = tiles > cus && rem > 0 && 2 * rem <= cus;
  if (split && cus % 8 == 0) {
    // Both parts in one launch of one workgroup per CU.
    const RoundsArgs r{g, tiles - rem};
    if (g.K % kTK != 0)
      hipLaunchKernelGGL((gemm_rounds_kernel<true>), dim3((unsigned)cus), dim3(kThreads), 0,
                         stream, r);
    else
      hipLaunchKernelGGL((gemm_rounds_kernel<false>), dim3((unsigned)cus), dim3(kThreads), 0,
                         stream, r);
    return hipGetLastError();
  }
  GemmArgs full = g;
  full.tile0 = 0;
  launch_part<kTM>(full, split ? tiles - rem : tiles, stream);
  if (split) {
    GemmArgs part = g;
    part.tile0 = tiles - rem;
    launch_part<128>(part, 2 * rem, stream);
  }
  return hipGetLastError();
}

}  // namespace attn
