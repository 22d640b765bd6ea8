// Fused attention backward for gfx950.
//
// With P recomputed from the forward's log-sum-exp L (P_ij = exp(scale
// q_i.k_j - L_i)) and Delta_i = sum_d dO_id O_id, the gradients of
// sum(dO * O) are
//   dV = P^T dO,  dP = dO V^T,  dS = P * (dP - Delta),  dQ = scale dS K,
//   dK = scale dS^T Q
// (the backward workloads of PTXBench, Appendix A, consume Q, K, V, O, dO and
// L and return dQ, dK, dV).  Two kernels, both free of atomics:
//
//  * bwd_dq_kernel: one workgroup of 4 wavefronts per (segment, query head,
//    128-row query block; the blocks with the most key tiles first), 32 rows
//    per wavefront, two workgroups per CU.  Its prologue computes Delta for its rows (the rows'
//    dO and O are read once) and stores -Delta, with L log2(e), in the
//    workspace (the dK/dV kernels start their dP accumulators from -Delta); the loop over key tiles recomputes S^T = K Q^T and
//    dP^T = V dO^T, forms dS^T in registers and accumulates dQ^T += K^T dS^T.
//  * bwd_dkdv_kernel / bwd_dkdv4_kernel: one workgroup per (segment,
//    key/value head, 128 keys), launched after bwd_dq_kernel (they read the
//    workspace).  The workgroup keeps its keys' K and V rows on chip (LDS,
//    or K in registers) and loops over every query head of the group and
//    every query tile that can see its keys, accumulating dV^T += dO^T P and
//    dK^T += Q^T dS in registers; the grouped-query sum therefore needs no
//    cross-workgroup reduction.  bwd_dkdv4_kernel has 4 wavefronts and two
//    workgroups per CU; at D = 128 and 96, causal grids too small for two
//    rounds of it use bwd_dkdv_kernel, with 8 wavefronts and one workgroup
//    per CU (see dkdv_form_for).
//
// Tiles of 64 rows (K and V for dQ; Q, dO, L log2 e and -Delta for dK/dV, in
// 32-row steps for bwd_dkdv4_kernel) go from global memory straight into a
// ring of LDS stages (buffer_load ... lds,
// bounded at the segment end so that rows past it read as zero), issued a
// tile ahead with one barrier per tile.  They stay row-major in LDS: operands
// whose reduction index runs along the tile's rows (K^T, Q^T, dO^T) come out
// of the same tiles through the transposing read ds_read_b64_tr_b16.
// Accumulator tiles are fed back as B operands directly (device_common.hpp).
//
// The backward expects a finite L for every row that has a visible key (as
// the forward produces); rows past the segment end read L = Delta = 0 and
// contribute nothing, because their dO rows read as zero.
#include <type_traits>

#include "attn_kernels.hpp"
#include "device_common.hpp"

namespace attn {
namespace {

constexpr int kTileRows = 64;

// The query-side rows that a dK/dV workgroup copies, pair by pair of its
// loop: pair n is query head g = n / per_head of the group and step
// j = n % per_head, whose rows start at (it0 + per_head - 1 - j) ROWS (the
// steps of a head are walked from the last down).  The walk holds j and the
// current head's row-0 pointers and moves them by addition, so the loop
// needs no division and no 64-bit products.  A row of a q-like tensor is
// below 2^24 bytes (128 rows are below 2^31, which the API checks), so row
// offsets are 32-bit products, and each descriptor covers the rows from its
// step to the segment end (row0 < len always), capped at whole rows below
// 2^31 bytes.
template <int ROWS>
struct QueryWalk {
  const char* q;      // the current head's row 0 (segment start)
  const char* dout;
  const char* lse;
  const char* del;
  int64_t q_head_b, r_head_b;   // bytes from one query head to the next
  int row_b, cap_rows, len, top, per_head;
  int j = 0;
  static constexpr int kCap4 = 0x7fffffff / 4;
  __device__ __forceinline__ int row0() const { return top - j * ROWS; }
  __device__ __forceinline__ i32x4 q_desc() const {
    return rows_desc_rb(q, row0(), len, row_b, cap_rows);
  }
  __device__ __forceinline__ i32x4 dout_desc() const {
    return rows_desc_rb(dout, row0(), len, row_b, cap_rows);
  }
  __device__ __forceinline__ i32x4 lse_desc() const { return rows_desc_rb(lse, row0(), len, 4, kCap4); }
  __device__ __forceinline__ i32x4 del_desc() const { return rows_desc_rb(del, row0(), len, 4, kCap4); }
  __device__ __forceinline__ void next() {
    if (++j == per_head) {
      j = 0;
      q += q_head_b;
      dout += q_head_b;
      lse += r_head_b;
      del += r_head_b;
    }
  }
};

template <int ROWS>
__device__ __forceinline__ QueryWalk<ROWS> query_walk(const BwdArgs& a, int64_t qseg,
                                                      int64_t rseg, int hk, int len, int it0,
                                                      int per_head) {
  QueryWalk<ROWS> w;
  const Layout& L = a.L;
  const int64_t h0 = (int64_t)hk * L.group;
  w.q = reinterpret_cast<const char*>(a.q + qseg + h0 * L.q_head);
  w.dout = reinterpret_cast<const char*>(a.dout + qseg + h0 * L.q_head);
  w.lse = reinterpret_cast<const char*>(a.lse2 + rseg + h0 * L.r_head);
  w.del = reinterpret_cast<const char*>(a.delta + rseg + h0 * L.r_head);
  w.q_head_b = L.q_head * 2;
  w.r_head_b = L.r_head * 4;
  w.row_b = (int)(L.q_row * 2);
  w.cap_rows = 0x7fffffff / w.row_b;
  w.len = len;
  w.top = (it0 + per_head - 1) * ROWS;
  w.per_head = per_head;
  return w;
}

// ---------------------------------------------------------------------------
// dQ (and Delta)
//
// Four wavefronts per workgroup of 128 query rows, 32 rows each, and two
// workgroups per CU (within 256 VGPRs per wavefront and 64 KiB of LDS per
// workgroup): the two wavefronts on a SIMD belong to different workgroups,
// so no common barrier holds them in step, and one workgroup's prologue and
// epilogue run under the other's loop.  K and V tiles stream through two
// LDS stages; each wavefront takes both 32-key halves of every tile.  The
// query blocks with the most key tiles under the causal mask go first.
// ---------------------------------------------------------------------------
constexpr int kQM = 128;   // query rows per workgroup
constexpr int kDqWaves = 4;
constexpr int kDqThreads = 64 * kDqWaves;

template <int D>
struct DqSmem {
  static constexpr int P = lds_pitch<D>();  // LDS row pitch (elements)
  static constexpr int TILE = 64 * P * 2;   // bytes of a 64-row bf16 tile
  static constexpr int K = 0;               // 2 stages
  static constexpr int V = K + 2 * TILE;    // 2 stages
  static constexpr int BYTES = V + 2 * TILE;
  static_assert(kDqWaves * 32 * P * 2 <= BYTES, "epilogue staging");
};

template <int D, bool CAUSAL>
__global__ __launch_bounds__(kDqThreads, 2) void bwd_dq_kernel(BwdArgs a) {
  using Tile = AsyncTile<D, kDqWaves>;
  using SM = DqSmem<D>;
  constexpr int P = SM::P;
  __shared__ __attribute__((aligned(1024))) char smem[SM::BYTES];

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = wave_id();
  const int l32 = lane & 31, half = lane >> 5;

  const Layout L = a.L;
  int gk, j, p;
  if (!xcd_decode((int)blockIdx.x, a.xo, gk, j, p)) return;
  const int z = gk / L.Hkv;
  const int h = (gk % L.Hkv) * L.group + j;
  const int hk = h / L.group;
  const Segment seg = segment_of(L, z);
  const int nqt = (seg.len + kQM - 1) / kQM;
  if (p >= nqt) return;

  // Fields used inside the lambdas below, as plain values (capturing the
  // kernel argument itself would make the compiler spill it to scratch).
  const int len = seg.len;
  const float sl2 = a.scale_log2;
  const float scale = a.scale;
  const int kv_rb = (int)(L.kv_row * 2);   // below 2^24: k-like rows are no wider than q-like
  const int kv_cap = 0x7fffffff / kv_rb;
  const int64_t q_row = L.q_row;
  const uint32_t sbase = lds_addr(smem);
  const Tile dma(wave, lane, kv_rb);
  const RowReader<D> rr(l32, half);
  const TransReader<D> trr(lane);

  {
    const int qt = nqt - 1 - p;
    const int q0 = qt * kQM;
    const int64_t qoff = (int64_t)seg.start * L.q_row + (int64_t)z * L.q_batch +
                         (int64_t)h * L.q_head;
    const int64_t kvoff = (int64_t)seg.start * L.kv_row + (int64_t)z * L.kv_batch +
                          (int64_t)hk * L.kv_head;
    const int64_t roff = (int64_t)seg.start + (int64_t)z * L.r_batch + (int64_t)h * L.r_head;
    const char* const kp = reinterpret_cast<const char*>(a.k + kvoff);
    const char* const vp = reinterpret_cast<const char*>(a.v + kvoff);

    const int qw0 = q0 + wave * 32;
    const int qrow = qw0 + l32;
    const bool valid = qrow < len;

    const int kend = CAUSAL ? min(len, q0 + kQM) : len;
    const int nkt = (kend + kTileRows - 1) / kTileRows;
    auto issue = [&](int kt) __attribute__((always_inline)) {
      const uint32_t st = (uint32_t)(kt & 1) * SM::TILE;
      // kt < nkt, so the tile starts before the segment end.
      dma_tile<D>(dma, rows_desc_rb(kp, kt * kTileRows, len, kv_rb, kv_cap), sbase + SM::K + st,
                  wave);
      dma_tile<D>(dma, rows_desc_rb(vp, kt * kTileRows, len, kv_rb, kv_cap), sbase + SM::V + st,
                  wave);
    };
    // Both stages are free: the first two tiles go out before the row loads.
    issue(0);
    if (nkt > 1) issue(1);

    // Q^T and dO^T as B operands; Delta from dO and O in the same layout.
    u32x4 qreg[D / 16], doreg[D / 16];
    float dsum = 0.f, lse2 = 0.f;
    {
      const rsrc_t rq = rows_rsrc(a.q + qoff, qw0, len, q_row);
      const rsrc_t rdo = rows_rsrc(a.dout + qoff, qw0, len, q_row);
      const rsrc_t ro = rows_rsrc(a.o + qoff, qw0, len, q_row);
      const int base = l32 * (int)(q_row * 2) + 16 * half;
      u32x4 ov[D / 16];
#pragma unroll
      for (int c = 0; c < D / 16; ++c) {
        qreg[c] = bload16(rq, base + 32 * c);
        doreg[c] = bload16(rdo, base + 32 * c);
        ov[c] = bload16(ro, base + 32 * c);
      }
      if (valid) lse2 = a.lse[roff + qrow] * kLog2e;
      // Every row load is in flight before the first use.
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int c = 0; c < D / 16; ++c)
#pragma unroll
        for (int w = 0; w < 4; ++w)
          dsum += bf16_lo(doreg[c][w]) * bf16_lo(ov[c][w]) + bf16_hi(doreg[c][w]) * bf16_hi(ov[c][w]);
    }
    const float delta = sum_halves(dsum);
    if (valid && half == 0) {
      a.delta[roff + qrow] = -delta;   // negated: the dK/dV kernels start dP from it
      a.lse2[roff + qrow] = lse2;
    }

    f32x16 dqacc[D / 32];
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
      for (int r = 0; r < 16; ++r) dqacc[db][r] = 0.f;
    // At D = 128 the dP^T products start from -Delta of the lane's row, held
    // in every element of a loop-invariant tile (the MFMA's accumulator
    // input), so that they give dP^T - Delta with no subtraction (32 vector
    // instructions per tile).  At D = 96 the tile's 16 registers cost more
    // than that (measured), and D = 64 gains nothing; there dP^T starts from
    // 0 and Delta is subtracted.
    constexpr bool kDeltaInit = D == 128;
    f32x16 ndelta;
#pragma unroll
    for (int r = 0; r < 16; ++r) ndelta[r] = kDeltaInit ? -delta : 0.f;

    // One tile, one 32-key half kb at a time (32 keys x 32 rows):
    //   S^T = K Q^T and dP^T = V dO^T (MFMA);
    //   P^T = exp2(s scale log2 e - L log2 e), masked only on tiles at the
    //   causal diagonal or the sequence end, and dS^T = P^T (dP^T - Delta),
    //   packed to bf16 (VALU);
    //   dQ^T += K^T dS^T with K^T read transposed (MFMA).
    auto compute = [&](int kt, auto masked) __attribute__((always_inline)) {
      const uint32_t st = (uint32_t)(kt & 1) * SM::TILE;
      const uint16_t* kc = reinterpret_cast<const uint16_t*>(smem + SM::K + st);
      const uint16_t* vc = reinterpret_cast<const uint16_t*>(smem + SM::V + st);
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        const int ks0 = kt * kTileRows + 32 * kb;
        // Under the causal mask a half whose first key follows the last row
        // contributes nothing.
        if constexpr (CAUSAL && decltype(masked)::value)
          if (ks0 > qw0 + 31) continue;
        f32x16 s, dp = ndelta;
#pragma unroll
        for (int r = 0; r < 16; ++r) s[r] = 0.f;
#pragma unroll
        for (int c = 0; c < D / 16; ++c) {
          const int o = rr.rm[c] + 32 * kb * P;
          s = mfma32(ld16(kc + o), qreg[c], s);
          dp = mfma32(ld16(vc + o), doreg[c], dp);
        }
        // s[r]: key ks0 + 8(r/4) + 4half + r%4, query qrow.
        const int t = ks0 + 4 * half - qrow;   // the lane's first key minus its query
        const int u = ks0 + 4 * half - len;    // the lane's first key minus the end
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          float pe = fast_exp2(__builtin_fmaf(s[r], sl2, -lse2));
          if constexpr (decltype(masked)::value) {
            const int off = 8 * (r / 4) + (r % 4);
            if constexpr (CAUSAL) pe = t + off > 0 ? 0.f : pe;   // key after query
            pe = u + off >= 0 ? 0.f : pe;                        // key past the end
          }
          s[r] = kDeltaInit ? pe * dp[r] : pe * (dp[r] - delta);
        }
#pragma unroll
        for (int c = 0; c < 2; ++c) {
          const u32x4 b = pack_chunk(s, c);
          const int rc = 16 * (2 * kb + c) * P;
#pragma unroll
          for (int db = 0; db < D / 32; ++db) {
            const u32x2 lo = ld_tr(kc + trr.tr[db][0] + rc), hi = ld_tr(kc + trr.tr[db][1] + rc);
            dqacc[db] = mfma32(u32x4{lo[0], lo[1], hi[0], hi[1]}, b, dqacc[db]);
          }
        }
      }
    };

    // Tile kt: wait for this wavefront's copies of it, then the barrier makes
    // every wavefront's share visible and frees the other stage (tile kt - 1),
    // which tile kt + 1 now fills (tile 1 went out with tile 0).
    int kt = 0;
    auto sync = [&]() __attribute__((always_inline)) {
      if (kt == 0 && nkt > 1)
        wait_vm_upto<2 * Tile::NJ>();
      else
        wait_vm_all();
      __syncthreads();
      if (kt > 0 && kt + 1 < nkt) issue(kt + 1);
    };
    // Key tiles past this wavefront's last row are fully masked for it.
    const int nkt_w = qw0 >= len ? 0 : CAUSAL ? min(nkt, (qw0 + 31) / kTileRows + 1) : nkt;
    // Tiles [0, nkt_u) need no mask for any of the wavefront's rows.
    const int nkt_u = min(nkt_w, CAUSAL ? min((qw0 + 1) / kTileRows, len / kTileRows)
                                        : len / kTileRows);
    while (kt < nkt_u) {
      sync();
      compute(kt, std::false_type{});
      ++kt;
    }
    while (kt < nkt_w) {
      sync();
      compute(kt, std::true_type{});
      ++kt;
    }
    while (kt < nkt) {   // fully masked for this wavefront: loads only
      sync();
      ++kt;
    }

    // Epilogue: scaled dQ rows staged as bf16 in LDS (this wavefront's own
    // region, 16-byte chunks swizzled by row), then written out as whole
    // rows (coalesced 16-byte stores).
    __syncthreads();   // every wavefront is done with the stages
    uint16_t* stg = reinterpret_cast<uint16_t*>(smem + wave * 32 * P * 2);
    const int sw = tile_swz<P>(l32);
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const f32x16& v = dqacc[db];
        st8(stg + l32 * P + 8 * ((4 * db + g) ^ sw) + 4 * half,
            u32x2{pack_bf16(v[4 * g] * scale, v[4 * g + 1] * scale),
                  pack_bf16(v[4 * g + 2] * scale, v[4 * g + 3] * scale)});
      }
    constexpr int CPR = D / 8;
    uint16_t* const dqp = a.dq + qoff;
#pragma unroll
    for (int i = 0; i < 32 * CPR / 64; ++i) {
      const int pidx = i * 64 + lane;
      const int row = pidx / CPR, ch = pidx % CPR;
      const u32x4 v = ld16(stg + row * P + 8 * (ch ^ tile_swz<P>(row)));
      if (qw0 + row < len) st16(dqp + (int64_t)(qw0 + row) * q_row + 8 * ch, v);
    }
  }
}

// ---------------------------------------------------------------------------
// dK, dV
//
// The eight-wavefront form (D = 128 and 96, rows padded to 128 elements in
// LDS; used for causal grids too small for two rounds of the four-wavefront
// form below).  A workgroup covers 128 keys, 32 per wavefront group.  K and
// V of the workgroup's keys stay in LDS (read as B operands) and the
// query-side tiles (Q, dO, L log2 e, Delta) stream through two LDS stages.
// Wavefronts w and w + 4 (which share a SIMD) own the same 32 keys and take
// the two 32-query halves of every 64-query tile, and their two partial
// dK/dV accumulators are added through LDS at the end (one workgroup per
// CU: 129 KiB of LDS).
// ---------------------------------------------------------------------------
constexpr int kKN = 128;        // keys per workgroup
constexpr int kDkvWaves = 8;

template <int D>
struct DkvSmem {
  static constexpr int P = lds_pitch<D>();                 // LDS row pitch (elements)
  static constexpr int TILE = 64 * P * 2;                  // bytes of a 64-row bf16 tile
  static constexpr int K = 0;                              // 2 tiles: keys 0-63, 64-127
  static constexpr int V = K + 2 * TILE;
  static constexpr int Q = V + 2 * TILE;                   // 2 stages
  static constexpr int DO = Q + 2 * TILE;                  // 2 stages
  static constexpr int LSE = DO + 2 * TILE;                // 2 stages x 64 fp32
  static constexpr int DEL = LSE + 2 * 256;
  static constexpr int BYTES = DEL + 2 * 256;
  // epilogue: one tensor's fp32 partial per wavefront
  static_assert(kDkvWaves * (D / 32) * 4 * 1024 <= BYTES, "reduction buffer");
};

template <int D, bool CAUSAL>
__global__ __launch_bounds__(64 * kDkvWaves, 1) void bwd_dkdv_kernel(BwdArgs a) {
  static_assert(D != 64, "D = 64 has the four-wavefront form only");
  constexpr int NW = kDkvWaves;
  using Tile = AsyncTile<D, NW>;
  using SM = DkvSmem<D>;
  constexpr int P = SM::P;
  __shared__ __attribute__((aligned(1024))) char smem[SM::BYTES];
  uint16_t* const sk = reinterpret_cast<uint16_t*>(smem + SM::K);
  uint16_t* const sv = reinterpret_cast<uint16_t*>(smem + SM::V);

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = wave_id();
  const int l32 = lane & 31, half = lane >> 5;
  const int kq = wave & 3;            // 32-key group
  const int sb = wave >> 2;   // query half of each tile

  const Layout L = a.L;
  int gk, j0, kb;
  if (!xcd_decode((int)blockIdx.x, a.xk, gk, j0, kb)) return;
  (void)j0;   // one head per group
  const int z = gk / L.Hkv, hk = gk % L.Hkv;
  const Segment seg = segment_of(L, z);
  const int k0 = kb * kKN;   // lowest keys (most work) first
  if (k0 >= seg.len) return;

  const int64_t kvoff = (int64_t)seg.start * L.kv_row + (int64_t)z * L.kv_batch +
                        (int64_t)hk * L.kv_head;
  const int64_t qseg = (int64_t)seg.start * L.q_row + (int64_t)z * L.q_batch;
  const int64_t rseg = (int64_t)seg.start + (int64_t)z * L.r_batch;

  const int kw0 = k0 + kq * 32;
  const int krow = kw0 + l32;
  // Fields used inside the lambdas below, as plain values (capturing the
  // kernel argument itself would make the compiler spill it to scratch).
  const int group = L.group;
  const int len = seg.len;
  const float sl2 = a.scale_log2;

  // Iterations run over (group head g, query tile it) with it from the first
  // tile that can see key k0.
  const int it0 = CAUSAL ? k0 / kTileRows : 0;
  const int nqt = (seg.len + kTileRows - 1) / kTileRows;
  const int per_head = nqt - it0;
  const int niter = per_head * L.group;
  const int top = (it0 + per_head - 1) * kTileRows;   // first row of each head's first tile
  // Q, dO, L log2(e) (written by the dQ kernel) and -Delta rows of the tiles.
  QueryWalk<kTileRows> walk = query_walk<kTileRows>(a, qseg, rseg, hk, len, it0, per_head);

  const Tile qdma(wave, lane, (int)(L.q_row * 2));
  const RowReader<D> rr(l32, half);
  const TransReader<D> trr(lane);
  const uint32_t sbase = lds_addr(smem);

  // K and V rows of the workgroup (once).
  {
    const Tile kvdma(wave, lane, (int)(L.kv_row * 2));
    const int64_t kv_row_b = L.kv_row * 2;
#pragma unroll
    for (int t = 0; t < 2; ++t) {
      dma_tile<D>(kvdma, rows_desc(a.k + kvoff, k0 + 64 * t, len, kv_row_b),
                  sbase + SM::K + t * SM::TILE, wave);
      dma_tile<D>(kvdma, rows_desc(a.v + kvoff, k0 + 64 * t, len, kv_row_b),
                  sbase + SM::V + t * SM::TILE, wave);
    }
  }

  // Copies of the walk's next tile into stage st.
  auto issue = [&](int st) __attribute__((always_inline)) {
    dma_tile<D>(qdma, walk.q_desc(), sbase + SM::Q + st * SM::TILE, wave);
    dma_tile<D>(qdma, walk.dout_desc(), sbase + SM::DO + st * SM::TILE, wave);
    if (wave == 0 && lane < 16) {
      dma16(walk.lse_desc(), sbase + SM::LSE + st * 256, 16 * lane);
      dma16(walk.del_desc(), sbase + SM::DEL + st * 256, 16 * lane);
    }
    walk.next();
  };

  f32x16 dkacc[D / 32], dvacc[D / 32];
#pragma unroll
  for (int db = 0; db < D / 32; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      dkacc[db][r] = 0.f;
      dvacc[db][r] = 0.f;
    }

  // This wavefront's K and V rows: tile kq / 2, rows 32 (kq % 2) + l32.
  const uint16_t* const krd = sk + (kq >> 1) * (SM::TILE / 2) + 32 * (kq & 1) * P;
  const uint16_t* const vrd = sv + (kq >> 1) * (SM::TILE / 2) + 32 * (kq & 1) * P;

  // Query half hq (32 queries) of the tile whose first row is qt0, in stage
  // st, against this wavefront's 32 keys.
  auto compute = [&](int qt0, int st, int hq, auto masked) __attribute__((always_inline)) {
    const uint16_t* q = reinterpret_cast<const uint16_t*>(smem + SM::Q + st * SM::TILE);
    const uint16_t* dout = reinterpret_cast<const uint16_t*>(smem + SM::DO + st * SM::TILE);
    const float* lse = reinterpret_cast<const float*>(smem + SM::LSE + st * 256);
    const float* del = reinterpret_cast<const float*>(smem + SM::DEL + st * 256);
    const int qs0 = qt0 + 32 * hq;
    // S = Q K^T, dP - Delta = dO V^T - Delta for this wavefront's 32 queries
    // x 32 keys: dP starts from the workspace's -Delta of each element's
    // query (s[r], dp[r]: query qs0 + 8(r/4) + 4half + r%4, key krow).
    f32x16 s, dp;
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const f32x4 nd4 = *reinterpret_cast<const f32x4*>(&del[32 * hq + 8 * g + 4 * half]);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        s[4 * g + i] = 0.f;
        dp[4 * g + i] = nd4[i];
      }
    }
#pragma unroll
    for (int c = 0; c < D / 16; ++c) {
      const int o = rr.rm[c] + 32 * hq * P;
      s = mfma32(ld16(q + o), ld16(krd + rr.rm[c]), s);
      dp = mfma32(ld16(dout + o), ld16(vrd + rr.rm[c]), dp);
    }
    // The first half of the L log2(e) values, then the transposed operands
    // of the first dV and dK products, whose latency the softmax covers (LDS
    // reads complete in order).
    const int rc0 = 16 * (2 * hq) * P;
    const f32x4 l4a = *reinterpret_cast<const f32x4*>(&lse[32 * hq + 4 * half]);
    const f32x4 l4b = *reinterpret_cast<const f32x4*>(&lse[32 * hq + 8 + 4 * half]);
    __builtin_amdgcn_sched_barrier(0);
    const u32x2 dlo0 = ld_tr(dout + trr.tr[0][0] + rc0), dhi0 = ld_tr(dout + trr.tr[0][1] + rc0);
    const u32x2 qlo0 = ld_tr(q + trr.tr[0][0] + rc0), qhi0 = ld_tr(q + trr.tr[0][1] + rc0);
    __builtin_amdgcn_sched_barrier(0);
    const int t = krow - qs0 - 4 * half;   // key minus the lane's first query
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const f32x4 l4 = g == 0 ? l4a : g == 1 ? l4b
                              : *reinterpret_cast<const f32x4*>(&lse[32 * hq + 8 * g + 4 * half]);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int r = 4 * g + i;
        float p = fast_exp2(__builtin_fmaf(s[r], sl2, -l4[i]));
        if constexpr (decltype(masked)::value) p = t > 8 * g + i ? 0.f : p;   // key after query
        s[r] = p;
        dp[r] = p * dp[r];
      }
    }
    // dV^T[d][key] += sum_q dO^T[d][q] P[q][key];  dK^T += Q^T dS, with the
    // A operands read transposed out of the row-major dO and Q tiles.
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      const u32x4 pb = pack_chunk(s, c);
      const u32x4 dsb = pack_chunk(dp, c);
      const int rc = 16 * (2 * hq + c) * P;
#pragma unroll
      for (int db = 0; db < D / 32; ++db) {
        const bool pre = c == 0 && db == 0;
        const u32x2 dlo = pre ? dlo0 : ld_tr(dout + trr.tr[db][0] + rc);
        const u32x2 dhi = pre ? dhi0 : ld_tr(dout + trr.tr[db][1] + rc);
        dvacc[db] = mfma32(u32x4{dlo[0], dlo[1], dhi[0], dhi[1]}, pb, dvacc[db]);
        const u32x2 qlo = pre ? qlo0 : ld_tr(q + trr.tr[db][0] + rc);
        const u32x2 qhi = pre ? qhi0 : ld_tr(q + trr.tr[db][1] + rc);
        dkacc[db] = mfma32(u32x4{qlo[0], qlo[1], qhi[0], qhi[1]}, dsb, dkacc[db]);
      }
    }
  };

  // Tile n has landed for this wavefront once its DMAs are done; the barrier
  // makes every wavefront's share visible and frees the stage read at n - 1,
  // which the loads of tile n + 1 now fill.  Only the first two query tiles
  // of each head (those reaching below the causal diagonal of this
  // workgroup's keys) are masked; rows past the end need no mask, as their
  // Q and dO read as zero.
  // Step n, the tile of head n / per_head whose first row is qt0.
  auto step = [&](int n, int qt0, auto masked) __attribute__((always_inline)) {
    wait_vm_all();
    __syncthreads();
    if (n + 1 < niter) issue((n + 1) & 1);
    compute(qt0, n & 1, sb, masked);
  };
  // Each head's query tiles are walked from the last down to the diagonal,
  // so that the workgroups of one key/value head (all starting with the
  // head's last tiles) read the same Q and dO tiles at about the same time
  // and share them in their XCD's L2; the two masked tiles come last.
  const int nmask = CAUSAL ? min(2, per_head) : 0;
  issue(0);
  int n = 0;
  for (int g = 0; g < group; ++g) {
    const int nend = n + per_head;
    int qt0 = top;
    for (const int nu = nend - nmask; n < nu; ++n, qt0 -= kTileRows)
      step(n, qt0, std::false_type{});
    for (; n < nend; ++n, qt0 -= kTileRows) step(n, qt0, std::true_type{});
  }

  // Epilogue.  Rows are staged as bf16 in LDS ([32 keys][D], 16-byte chunks
  // swizzled by row as in the tiles) and written out as whole rows
  // (coalesced 16-byte stores).
  __syncthreads();   // every wavefront is done with the tiles
  const int64_t kv_row = L.kv_row;
  auto store_rows = [&](const f32x16 (&acc)[D / 32], float mul, uint16_t* stg, uint16_t* gout)
      __attribute__((always_inline)) {
    const int sw = tile_swz<P>(l32);
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
      for (int g = 0; g < 4; ++g)
        st8(stg + l32 * P + 8 * ((4 * db + g) ^ sw) + 4 * half,
            u32x2{pack_bf16(acc[db][4 * g] * mul, acc[db][4 * g + 1] * mul),
                  pack_bf16(acc[db][4 * g + 2] * mul, acc[db][4 * g + 3] * mul)});
    constexpr int CPR = D / 8;
#pragma unroll
    for (int i = 0; i < 32 * CPR / 64; ++i) {
      const int pidx = i * 64 + lane;
      const int row = pidx / CPR, ch = pidx % CPR;
      const u32x4 v = ld16(stg + row * P + 8 * (ch ^ tile_swz<P>(row)));
      if (kw0 + row < len) st16(gout + (int64_t)(kw0 + row) * kv_row + 8 * ch, v);
    }
  };
  {
    // The pair splits the work: the sb = 0 wavefront finalises dK, the
    // sb = 1 one dV.  Each first hands its partial of the other tensor to
    // its partner, then adds the partner's partial to its own.
    u32x4* const red = reinterpret_cast<u32x4*>(smem);
    constexpr int SL = (D / 32) * 4;   // u32x4 slots per lane for one tensor
    auto hand = [&](const f32x16 (&acc)[D / 32]) __attribute__((always_inline)) {
#pragma unroll
      for (int db = 0; db < D / 32; ++db)
#pragma unroll
        for (int j = 0; j < 4; ++j)
          red[(wave * SL + 4 * db + j) * 64 + lane] =
              u32x4{__float_as_uint(acc[db][4 * j]), __float_as_uint(acc[db][4 * j + 1]),
                    __float_as_uint(acc[db][4 * j + 2]), __float_as_uint(acc[db][4 * j + 3])};
    };
    if (sb == 0)
      hand(dvacc);
    else
      hand(dkacc);
    __syncthreads();
    auto finalize = [&](f32x16 (&acc)[D / 32], float mul, uint16_t* gout) __attribute__((always_inline)) {
      const u32x4* src = red + (wave ^ 4) * SL * 64;
#pragma unroll
      for (int db = 0; db < D / 32; ++db)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const u32x4 pp = src[(4 * db + j) * 64 + lane];
#pragma unroll
          for (int i = 0; i < 4; ++i) acc[db][4 * j + i] += __uint_as_float(pp[i]);
        }
      // Staged in the partner's region, read above.
      store_rows(acc, mul, reinterpret_cast<uint16_t*>(red + (wave ^ 4) * SL * 64), gout);
    };
    if (sb == 0)
      finalize(dkacc, a.scale, a.dk + kvoff);
    else
      finalize(dvacc, 1.f, a.dv + kvoff);
  }
}

// ---------------------------------------------------------------------------
// dK, dV, four-wavefront form (every D; the only form at D = 64): four
// wavefronts per 128 keys, two workgroups per CU (three at D = 64, whose
// registers allow it).  Each wavefront owns 32 keys outright (no partial to combine): its
// K rows stay in registers as the B operand of S = Q K^T, the workgroup's V
// rows in LDS (B operand of dP = dO V^T), and the query side streams through
// two LDS stages of 32 rows.  64.5 KiB of LDS per workgroup, so the two
// wavefronts on a SIMD come from different workgroups.
// ---------------------------------------------------------------------------
constexpr int kQS = 32;   // query rows per step

template <int D>
struct Dkv4Smem {
  static constexpr int P = lds_pitch<D>();
  static constexpr int TILE = 64 * P * 2;   // bytes of a 64-row bf16 tile
  static constexpr int HT = kQS * P * 2;    // bytes of a 32-row bf16 tile
  static constexpr int V = 0;               // 2 tiles: keys 0-63, 64-127
  static constexpr int Q = V + 2 * TILE;    // 2 stages
  static constexpr int DO = Q + 2 * HT;     // 2 stages
  static constexpr int LSE = DO + 2 * HT;   // 2 stages x 32 fp32
  static constexpr int DEL = LSE + 2 * kQS * 4;
  static constexpr int BYTES = DEL + 2 * kQS * 4;
  static_assert(4 * 2 * 32 * P * 2 <= BYTES, "epilogue staging");
};

template <int D, bool CAUSAL>
__global__ __launch_bounds__(256, 2) void bwd_dkdv4_kernel(BwdArgs a) {
  using SM = Dkv4Smem<D>;
  constexpr int P = SM::P;
  using VTile = AsyncTile<D, 4>;   // a 64-row tile, four wavefronts
  using HTile = AsyncTile<D, 8>;   // wavefronts 0-3 of eight: rows 0-31 of a tile
  __shared__ __attribute__((aligned(1024))) char smem[SM::BYTES];
  const uint16_t* const sv = reinterpret_cast<const uint16_t*>(smem + SM::V);

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = wave_id();
  const int l32 = lane & 31, half = lane >> 5;
  const int kq = wave;   // 32-key group

  const Layout L = a.L;
  int gk, j0, kb;
  if (!xcd_decode((int)blockIdx.x, a.xk, gk, j0, kb)) return;
  (void)j0;   // one head per group
  const int z = gk / L.Hkv, hk = gk % L.Hkv;
  const Segment seg = segment_of(L, z);
  const int k0 = kb * kKN;   // lowest keys (most work) first
  if (k0 >= seg.len) return;

  const int64_t kvoff = (int64_t)seg.start * L.kv_row + (int64_t)z * L.kv_batch +
                        (int64_t)hk * L.kv_head;
  const int64_t qseg = (int64_t)seg.start * L.q_row + (int64_t)z * L.q_batch;
  const int64_t rseg = (int64_t)seg.start + (int64_t)z * L.r_batch;
  const int kw0 = k0 + 32 * kq;
  const int krow = kw0 + l32;
  const int group = L.group;
  const int len = seg.len;
  const float sl2 = a.scale_log2;

  // Steps run over (group head g, 32-query step j), from the step holding
  // key k0 (causal) to the segment end.
  const int it0 = CAUSAL ? k0 / kQS : 0;
  const int nqs = (seg.len + kQS - 1) / kQS;
  const int per_head = nqs - it0;
  const int niter = per_head * L.group;
  const int top = (it0 + per_head - 1) * kQS;   // first row of each head's first step
  QueryWalk<kQS> walk = query_walk<kQS>(a, qseg, rseg, hk, len, it0, per_head);

  const HTile qdma(wave, lane, (int)(L.q_row * 2));
  const RowReader<D> rr(l32, half);
  const TransReader<D> trr(lane);
  const uint32_t sbase = lds_addr(smem);

  // V rows of the workgroup into LDS (once); this wavefront's K rows into
  // registers: kreg[c] = K[krow][16 c + 8 half .. + 7] (zero past the end).
  {
    const VTile vdma(wave, lane, (int)(L.kv_row * 2));
    const int64_t kv_row_b = L.kv_row * 2;
#pragma unroll
    for (int t = 0; t < 2; ++t)
      dma_tile<D>(vdma, rows_desc(a.v + kvoff, k0 + 64 * t, len, kv_row_b),
                  sbase + SM::V + t * SM::TILE, wave);
  }
  u32x4 kreg[D / 16];
  {
    const rsrc_t rk = rows_rsrc(a.k + kvoff, kw0, len, L.kv_row);
    const int base = l32 * (int)(L.kv_row * 2) + 16 * half;
#pragma unroll
    for (int c = 0; c < D / 16; ++c) kreg[c] = bload16(rk, base + 32 * c);
  }

  // Copies of the walk's next step into stage st.
  auto issue = [&](int st) __attribute__((always_inline)) {
    dma_tile<D>(qdma, walk.q_desc(), sbase + SM::Q + st * SM::HT, wave);
    dma_tile<D>(qdma, walk.dout_desc(), sbase + SM::DO + st * SM::HT, wave);
    if (wave == 0 && lane < 8) {
      dma16(walk.lse_desc(), sbase + SM::LSE + st * (kQS * 4), 16 * lane);
      dma16(walk.del_desc(), sbase + SM::DEL + st * (kQS * 4), 16 * lane);
    }
    walk.next();
  };

  f32x16 dkacc[D / 32], dvacc[D / 32];
#pragma unroll
  for (int db = 0; db < D / 32; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      dkacc[db][r] = 0.f;
      dvacc[db][r] = 0.f;
    }
  // This wavefront's V rows: tile kq / 2, rows 32 (kq % 2) + l32.
  const uint16_t* const vrd = sv + (kq >> 1) * (SM::TILE / 2) + 32 * (kq & 1) * P;

  // The 32 queries from qs0 (stage st) against this wavefront's 32 keys.
  auto compute = [&](int qs0, int st, auto masked) __attribute__((always_inline)) {
    const uint16_t* q = reinterpret_cast<const uint16_t*>(smem + SM::Q + st * SM::HT);
    const uint16_t* dout = reinterpret_cast<const uint16_t*>(smem + SM::DO + st * SM::HT);
    const float* lse = reinterpret_cast<const float*>(smem + SM::LSE + st * (kQS * 4));
    const float* del = reinterpret_cast<const float*>(smem + SM::DEL + st * (kQS * 4));
    // S = Q K^T and dP - Delta = dO V^T - Delta: dP starts from the
    // workspace's -Delta of each element's query (s[r], dp[r]: query
    // qs0 + 8(r/4) + 4half + r%4, key krow).
    f32x16 s, dp;
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const f32x4 nd4 = *reinterpret_cast<const f32x4*>(&del[8 * g + 4 * half]);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        s[4 * g + i] = 0.f;
        dp[4 * g + i] = nd4[i];
      }
    }
#pragma unroll
    for (int c = 0; c < D / 16; ++c) {
      s = mfma32(ld16(q + rr.rm[c]), kreg[c], s);
      dp = mfma32(ld16(dout + rr.rm[c]), ld16(vrd + rr.rm[c]), dp);
      // Keep at most four chunks of operands in flight (register budget).
      if (c % 4 == 3) __builtin_amdgcn_sched_barrier(0);
    }
    // The first half of the step's L log2(e) values, then the transposed
    // operands of the first dV and dK products (chunk 0, column block 0):
    // the softmax's vector work covers the latter's latency (LDS reads
    // complete in order, so they go out after the values the softmax
    // waits for first).
    const f32x4 l4a = *reinterpret_cast<const f32x4*>(&lse[4 * half]);
    const f32x4 l4b = *reinterpret_cast<const f32x4*>(&lse[8 + 4 * half]);
    __builtin_amdgcn_sched_barrier(0);
    const u32x2 dlo0 = ld_tr(dout + trr.tr[0][0]), dhi0 = ld_tr(dout + trr.tr[0][1]);
    const u32x2 qlo0 = ld_tr(q + trr.tr[0][0]), qhi0 = ld_tr(q + trr.tr[0][1]);
    __builtin_amdgcn_sched_barrier(0);
    const int t = krow - qs0 - 4 * half;   // key minus the lane's first query
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const f32x4 l4 = g == 0 ? l4a : g == 1 ? l4b
                              : *reinterpret_cast<const f32x4*>(&lse[8 * g + 4 * half]);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int r = 4 * g + i;
        float p = fast_exp2(__builtin_fmaf(s[r], sl2, -l4[i]));
        if constexpr (decltype(masked)::value) p = t > 8 * g + i ? 0.f : p;   // key after query
        s[r] = p;
        dp[r] = p * dp[r];
      }
    }
    // dV^T += dO^T P, dK^T += Q^T dS (A operands read transposed).
#pragma unroll
    for (int c = 0; c < 2; ++c) {
      const u32x4 pb = pack_chunk(s, c);
      const u32x4 dsb = pack_chunk(dp, c);
      const int rc = 16 * c * P;
#pragma unroll
      for (int db = 0; db < D / 32; ++db) {
        const bool pre = c == 0 && db == 0;
        const u32x2 dlo = pre ? dlo0 : ld_tr(dout + trr.tr[db][0] + rc);
        const u32x2 dhi = pre ? dhi0 : ld_tr(dout + trr.tr[db][1] + rc);
        dvacc[db] = mfma32(u32x4{dlo[0], dlo[1], dhi[0], dhi[1]}, pb, dvacc[db]);
        const u32x2 qlo = pre ? qlo0 : ld_tr(q + trr.tr[db][0] + rc);
        const u32x2 qhi = pre ? qhi0 : ld_tr(q + trr.tr[db][1] + rc);
        dkacc[db] = mfma32(u32x4{qlo[0], qlo[1], qhi[0], qhi[1]}, dsb, dkacc[db]);
      }
      __builtin_amdgcn_sched_barrier(0);
    }
  };

  // Step n: its copies have landed for this wavefront; the barrier makes
  // every wavefront's share visible and frees the stage read at n - 1, which
  // the copies of step n + 1 now fill.  Under the causal mask a wavefront
  // skips the steps whose queries all precede its keys and masks the one
  // holding its diagonal.
  auto sync = [&](int n) __attribute__((always_inline)) {
    wait_vm_all();
    __syncthreads();
    if (n + 1 < niter) issue((n + 1) & 1);
  };
  // Per head the query steps are walked from the last down to the
  // diagonal, so that the workgroups of one key/value head (all starting
  // with the head's last steps) read the same Q and dO rows at about the
  // same time and share them in their XCD's L2.  Under the causal mask the
  // last four steps hold the workgroup's diagonal (masked compute, skipped
  // by the wavefronts whose keys all follow the step's queries); the others
  // need no mask.  Each loop body has one form of compute (two forms in one
  // body exceed the register budget).
  const int ndiag = CAUSAL ? min(kKN / kQS, per_head) : 0;
  issue(0);
  // Wait for every load so far (K rows, V tile, step 0) through the builtin,
  // which the compiler's wait insertion sees (the first step waits for them
  // anyway).  Without it the compiler takes the K-row loads as possibly
  // outstanding inside the loop and puts vmcnt waits among the S products,
  // which then also wait for the next step's copies, issued just before.
  wait_vm<0>();
  int n = 0;
#pragma nounroll
  for (int g = 0; g < group; ++g) {
    int qs0 = top;   // first query of step n
#pragma nounroll
    for (const int nu = (g + 1) * per_head - ndiag; n < nu; ++n, qs0 -= kQS) {
      sync(n);
      compute(qs0, n & 1, std::false_type{});
    }
#pragma nounroll
    for (const int ne = (g + 1) * per_head; n < ne; ++n, qs0 -= kQS) {
      sync(n);
      if (qs0 >= kw0) compute(qs0, n & 1, std::true_type{});
    }
  }

  // Epilogue: each wavefront stages its bf16 dK and dV rows in LDS ([32
  // keys][D], 16-byte chunks swizzled by row) and writes whole rows.
  __syncthreads();   // every wavefront is done with the stages
  const int64_t kv_row = L.kv_row;
  auto store_rows = [&](const f32x16 (&acc)[D / 32], float mul, uint16_t* stg, uint16_t* gout)
      __attribute__((always_inline)) {
    const int sw = tile_swz<P>(l32);
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
      for (int g = 0; g < 4; ++g)
        st8(stg + l32 * P + 8 * ((4 * db + g) ^ sw) + 4 * half,
            u32x2{pack_bf16(acc[db][4 * g] * mul, acc[db][4 * g + 1] * mul),
                  pack_bf16(acc[db][4 * g + 2] * mul, acc[db][4 * g + 3] * mul)});
    constexpr int CPR = D / 8;
#pragma unroll
    for (int i = 0; i < 32 * CPR / 64; ++i) {
      const int pidx = i * 64 + lane;
      const int row = pidx / CPR, ch = pidx % CPR;
      const u32x4 v = ld16(stg + row * P + 8 * (ch ^ tile_swz<P>(row)));
      if (kw0 + row < len) st16(gout + (int64_t)(kw0 + row) * kv_row + 8 * ch, v);
    }
  };
  uint16_t* stg = reinterpret_cast<uint16_t*>(smem) + wave * 2 * 32 * P;
  store_rows(dkacc, a.scale, stg, a.dk + kvoff);
  store_rows(dvacc, 1.f, stg + 32 * P, a.dv + kvoff);
}

// Explicit instantiations: without them the host compiler may skip the
// launch stubs of these templates (leaving undefined symbols in the library).
template __global__ void bwd_dq_kernel<64, false>(BwdArgs);
template __global__ void bwd_dq_kernel<64, true>(BwdArgs);
template __global__ void bwd_dq_kernel<96, false>(BwdArgs);
template __global__ void bwd_dq_kernel<96, true>(BwdArgs);
template __global__ void bwd_dq_kernel<128, false>(BwdArgs);
template __global__ void bwd_dq_kernel<128, true>(BwdArgs);
template __global__ void bwd_dkdv_kernel<96, false>(BwdArgs);
template __global__ void bwd_dkdv_kernel<96, true>(BwdArgs);
template __global__ void bwd_dkdv_kernel<128, false>(BwdArgs);
template __global__ void bwd_dkdv_kernel<128, true>(BwdArgs);
template __global__ void bwd_dkdv4_kernel<64, false>(BwdArgs);
template __global__ void bwd_dkdv4_kernel<64, true>(BwdArgs);
template __global__ void bwd_dkdv4_kernel<96, false>(BwdArgs);
template __global__ void bwd_dkdv4_kernel<96, true>(BwdArgs);
template __global__ void bwd_dkdv4_kernel<128, false>(BwdArgs);
template __global__ void bwd_dkdv4_kernel<128, true>(BwdArgs);

}  // namespace

namespace {

template <int D>
void launch_bwd_d(const BwdArgs& a, int phases, hipStream_t stream) {
  // One dQ workgroup per query block (see the kernel), in the XCD-aware order.
  BwdArgs b = a;
  b.xo = xcd_order(a.L.nseg, a.L.Hkv, a.L.group, (a.L.S + kQM - 1) / kQM, a.causal != 0);
  b.xk = xcd_order(a.L.nseg, a.L.Hkv, 1, (a.L.S + kKN - 1) / kKN, a.causal != 0);
  const dim3 gq((unsigned)xcd_grid(b.xo));
  const dim3 gk((unsigned)xcd_grid(b.xk));
  if (phases & 1) {
    if (a.causal)
      hipLaunchKernelGGL((bwd_dq_kernel<D, true>), gq, dim3(kDqThreads), 0, stream, b);
    else
      hipLaunchKernelGGL((bwd_dq_kernel<D, false>), gq, dim3(kDqThreads), 0, stream, b);
  }
  if (phases & 2) {
    const int form = D == 64 ? 2
                     : a.dkdv_form ? a.dkdv_form
                                   : dkdv_form_for(a.L.nseg, a.L.Hkv, a.L.S, a.L.total,
                                                   a.L.cu != nullptr, D, a.causal != 0);
    if (form == 2) {
      if (a.causal)
        hipLaunchKernelGGL((bwd_dkdv4_kernel<D, true>), gk, dim3(256), 0, stream, b);
      else
        hipLaunchKernelGGL((bwd_dkdv4_kernel<D, false>), gk, dim3(256), 0, stream, b);
      return;
    }
    if constexpr (D != 64) {
      if (a.causal)
        hipLaunchKernelGGL((bwd_dkdv_kernel<D, true>), gk, dim3(64 * kDkvWaves), 0, stream, b);
      else
        hipLaunchKernelGGL((bwd_dkdv_kernel<D, false>), gk, dim3(64 * kDkvWaves), 0, stream, b);
    }
  }
}

}  // namespace

// Two workgroups per CU keep every workgroup of a grid resident from the
// start, so the unequal work of causal key blocks is only balanced (heaviest
// first) when there are at least two rounds of them; fewer go to the
// one-per-CU form.  Packed layouts count their sequences' blocks, about
// total / 128 + nseq per key head.
int dkdv_form_for(int nseg, int Hkv, int S, int total, bool packed, int D, bool causal) {
  if (D == 64) return 2;   // the four-wavefront form is the only one at D = 64
  const int64_t blocks = packed ? (int64_t)Hkv * (total / kKN + nseg)
                                : (int64_t)nseg * Hkv * ((S + kKN - 1) / kKN);
  return !causal || blocks >= 4 * kChipCUs ? 2 : 1;
}

hipError_t launch_bwd(const BwdArgs& a, int D, int phases, hipStream_t stream) {
  if (D == 64)
    launch_bwd_d<64>(a, phases, stream);
  else if (D == 96)
    launch_bwd_d<96>(a, phases, stream);
  else
    launch_bwd_d<128>(a, phases, stream);
  return hipGetLastError();
}

}  // namespace attn
