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
//  * bwd_dq_kernel: one workgroup per (segment, query head, 128 query rows),
//    32 rows per wavefront.  Its prologue computes Delta for its rows (the
//    rows' dO and O are read once) and stores it in the workspace; the loop
//    over key tiles recomputes S^T = K Q^T and dP^T = V dO^T, forms dS^T in
//    registers and accumulates dQ^T += K^T dS^T.
//  * bwd_dkdv_kernel: one workgroup per (segment, key/value head, 128 keys),
//    32 keys per wavefront, launched after bwd_dq_kernel (it reads Delta).
//    The wavefront keeps its K and V rows in registers and loops over every
//    query head of the group and every query tile that can see its keys,
//    accumulating dV^T += dO^T P and dK^T += Q^T dS in registers; the
//    grouped-query sum therefore needs no cross-workgroup reduction.
//
// Tiles of 64 rows (K and V for dQ; Q, dO, L and Delta for dK/dV) go from
// global memory straight into two LDS stages (buffer_load ... lds, bounded
// at the segment end so that rows past it read as zero), issued a tile ahead
// with one barrier per tile.  They stay row-major in LDS: operands whose
// reduction index runs along the tile's rows (K^T, Q^T, dO^T) come out of the
// same tiles through the transposing read ds_read_b64_tr_b16.  Accumulator
// tiles are fed back as B operands directly (device_common.hpp).
//
// The backward expects a finite L for every row that has a visible key (as
// the forward produces); rows past the segment end read L = Delta = 0 and
// contribute nothing, because their dO rows read as zero.
#include "attn_kernels.hpp"
#include "device_common.hpp"

namespace attn {
namespace {

constexpr int kThreads = 256;
constexpr int kTileRows = 64;

// Enqueue rows [row0, row0 + 64) of an fp32 row vector (L or Delta of one
// head) into a 256-byte LDS array: 16 lanes of one wavefront, 16 bytes each.
__device__ __forceinline__ void load_rowvec(const float* head_base, int row0, int len, float* dst,
                                            int lane) {
  if (lane < 16) {
    const rsrc_t r = make_rsrc(head_base + row0, (int64_t)(len - row0) * 4);
    __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (ATTN_LDS void*)dst, 16, 16 * lane, 0, 0, 0);
  }
}

// ---------------------------------------------------------------------------
// dQ (and Delta)
// ---------------------------------------------------------------------------
constexpr int kQM = 128;   // query rows per workgroup

template <int D>
__global__ __launch_bounds__(kThreads, 1) void bwd_dq_kernel(BwdArgs a) {
  using Tile = AsyncTile<D>;
  __shared__ __attribute__((aligned(1024))) uint16_t sk0[Tile::ELEMS];
  __shared__ __attribute__((aligned(1024))) uint16_t sk1[Tile::ELEMS];
  __shared__ __attribute__((aligned(1024))) uint16_t sv0[Tile::ELEMS];
  __shared__ __attribute__((aligned(1024))) uint16_t sv1[Tile::ELEMS];

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = wave_id();
  const int l32 = lane & 31, half = lane >> 5;

  const Layout L = a.L;
  const int z = blockIdx.x / L.Hq, h = blockIdx.x % L.Hq;
  const int hk = h / L.group;
  const Segment seg = segment_of(L, z);
  const int qt = (int)gridDim.y - 1 - (int)blockIdx.y;
  const int q0 = qt * kQM;
  if (q0 >= seg.len) return;

  const int64_t qoff = (int64_t)seg.start * L.q_row + (int64_t)z * L.q_batch +
                       (int64_t)h * L.q_head;
  const int64_t kvoff = (int64_t)seg.start * L.kv_row + (int64_t)z * L.kv_batch +
                        (int64_t)hk * L.kv_head;
  const int64_t roff = (int64_t)seg.start + (int64_t)z * L.r_batch + (int64_t)h * L.r_head;
  const uint16_t* kp = a.k + kvoff;
  const uint16_t* vp = a.v + kvoff;

  const int qw0 = q0 + wave * 32;
  const int qrow = qw0 + l32;
  const bool valid = qrow < seg.len;

  // Q^T and dO^T as B operands; Delta from dO and O in the same layout.
  u32x4 qreg[D / 16], doreg[D / 16];
  float dsum = 0.f;
  {
    const rsrc_t rq = rows_rsrc(a.q + qoff, qw0, seg.len, L.q_row);
    const rsrc_t rdo = rows_rsrc(a.dout + qoff, qw0, seg.len, L.q_row);
    const rsrc_t ro = rows_rsrc(a.o + qoff, qw0, seg.len, L.q_row);
    const int base = l32 * (int)(L.q_row * 2) + 16 * half;
#pragma unroll
    for (int c = 0; c < D / 16; ++c) {
      qreg[c] = bload16(rq, base + 32 * c);
      doreg[c] = bload16(rdo, base + 32 * c);
      const u32x4 ov = bload16(ro, base + 32 * c);
#pragma unroll
      for (int w = 0; w < 4; ++w)
        dsum += bf16_lo(doreg[c][w]) * bf16_lo(ov[w]) + bf16_hi(doreg[c][w]) * bf16_hi(ov[w]);
    }
  }
  const float delta = dsum + swap_halves(dsum);
  float lse2 = 0.f;
  if (valid) {
    lse2 = a.lse[roff + qrow] * kLog2e;
    if (half == 0) a.delta[roff + qrow] = delta;
  }

  const int kend = a.causal ? min(seg.len, q0 + kQM) : seg.len;
  const int nkt = (kend + kTileRows - 1) / kTileRows;
  // Key tiles past this wavefront's last query are fully masked for it.
  const int nkt_w = a.causal ? min(nkt, (qw0 + 31) / kTileRows + 1) : nkt;

  const Tile dma(wave, lane, (int)(L.kv_row * 2));
  const RowReader<D> rr(l32, half);
  const TransReader<D> trr(lane);
  const float sl2 = a.scale_log2;
  // Fields used inside the lambdas below, as plain values.
  const bool causal = a.causal != 0;
  const int len = seg.len;
  const int64_t kv_row = L.kv_row;

  f32x16 dqacc[D / 32];
#pragma unroll
  for (int db = 0; db < D / 32; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) dqacc[db][r] = 0.f;

  auto compute = [&](int kt, const uint16_t* kc, const uint16_t* vc) __attribute__((always_inline)) {
    const int k0 = kt * kTileRows;
    f32x16 s[2], dp[2];
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        s[kb][r] = 0.f;
        dp[kb][r] = 0.f;
      }
#pragma unroll
    for (int c = 0; c < D / 16; ++c)
#pragma unroll
      for (int kb = 0; kb < 2; ++kb) {
        const int o = rr.rm[c] + 32 * kb * D;
        s[kb] = mfma32(ld16(kc + o), qreg[c], s[kb]);
        dp[kb] = mfma32(ld16(vc + o), doreg[c], dp[kb]);
      }
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) s[kb][r] = fast_exp2(__builtin_fmaf(s[kb][r], sl2, -lse2));
    if ((causal && k0 + kTileRows - 1 > qw0) || k0 + kTileRows > len) {
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int key = k0 + 32 * kb + 8 * (r / 4) + 4 * half + (r % 4);
          s[kb][r] = ((causal && key > qrow) || key >= len) ? 0.f : s[kb][r];
        }
    }
#pragma unroll
    for (int kb = 0; kb < 2; ++kb)
#pragma unroll
      for (int r = 0; r < 16; ++r) s[kb][r] = s[kb][r] * (dp[kb][r] - delta);   // dS^T
    // dQ^T[d][q] += sum_key K^T[d][key] dS^T[key][q]; K^T read transposed.
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const u32x4 b = pack_chunk(s[c >> 1], c & 1);
#pragma unroll
      for (int db = 0; db < D / 32; ++db) {
        const u32x2 lo = ld_tr(kc + trr.tr[db][0] + 16 * c * D);
        const u32x2 hi = ld_tr(kc + trr.tr[db][1] + 16 * c * D);
        dqacc[db] = mfma32(u32x4{lo[0], lo[1], hi[0], hi[1]}, b, dqacc[db]);
      }
    }
  };
  auto step = [&](int kt, bool work, const uint16_t* kc, const uint16_t* vc, uint16_t* kn,
                  uint16_t* vn) __attribute__((always_inline)) {
    wait_vm<0>();
    __syncthreads();
    if (kt + 1 < nkt) {
      dma.load(rows_rsrc(kp, (kt + 1) * kTileRows, len, kv_row), kn, wave);
      dma.load(rows_rsrc(vp, (kt + 1) * kTileRows, len, kv_row), vn, wave);
    }
    if (work) compute(kt, kc, vc);
  };

  if (nkt > 0) {
    dma.load(rows_rsrc(kp, 0, seg.len, L.kv_row), sk0, wave);
    dma.load(rows_rsrc(vp, 0, seg.len, L.kv_row), sv0, wave);
  }
  wait_vm<0>();
  int kt = 0;
  for (; kt + 1 < nkt_w; kt += 2) {
    step(kt, true, sk0, sv0, sk1, sv1);
    step(kt + 1, true, sk1, sv1, sk0, sv0);
  }
  if (kt < nkt_w) {
    step(kt, true, sk0, sv0, sk1, sv1);
    ++kt;
  }
  for (; kt < nkt; ++kt) {
    if (kt & 1)
      step(kt, false, sk1, sv1, sk0, sv0);
    else
      step(kt, false, sk0, sv0, sk1, sv1);
  }

  if (valid) {
    uint16_t* dqp = a.dq + qoff + (int64_t)qrow * L.q_row;
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        u32x2 w;
        w[0] = pack_bf16(dqacc[db][4 * g + 0] * a.scale, dqacc[db][4 * g + 1] * a.scale);
        w[1] = pack_bf16(dqacc[db][4 * g + 2] * a.scale, dqacc[db][4 * g + 3] * a.scale);
        st8(dqp + 32 * db + 8 * g + 4 * half, w);
      }
  }
}

// ---------------------------------------------------------------------------
// dK, dV
// ---------------------------------------------------------------------------
constexpr int kKN = 128;   // keys per workgroup

template <int D>
__global__ __launch_bounds__(kThreads, 1) void bwd_dkdv_kernel(BwdArgs a) {
  using Tile = AsyncTile<D>;
  __shared__ __attribute__((aligned(1024))) uint16_t sq0[Tile::ELEMS];
  __shared__ __attribute__((aligned(1024))) uint16_t sq1[Tile::ELEMS];
  __shared__ __attribute__((aligned(1024))) uint16_t sdo0[Tile::ELEMS];
  __shared__ __attribute__((aligned(1024))) uint16_t sdo1[Tile::ELEMS];
  __shared__ __attribute__((aligned(16))) float sl0[kTileRows];
  __shared__ __attribute__((aligned(16))) float sl1[kTileRows];
  __shared__ __attribute__((aligned(16))) float sd0[kTileRows];
  __shared__ __attribute__((aligned(16))) float sd1[kTileRows];

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = wave_id();
  const int l32 = lane & 31, half = lane >> 5;

  const Layout L = a.L;
  const int z = blockIdx.x / L.Hkv, hk = blockIdx.x % L.Hkv;
  const Segment seg = segment_of(L, z);
  const int k0 = (int)blockIdx.y * kKN;   // lowest keys (most work) first
  if (k0 >= seg.len) return;

  const int64_t kvoff = (int64_t)seg.start * L.kv_row + (int64_t)z * L.kv_batch +
                        (int64_t)hk * L.kv_head;
  const int64_t qseg = (int64_t)seg.start * L.q_row + (int64_t)z * L.q_batch;
  const int64_t rseg = (int64_t)seg.start + (int64_t)z * L.r_batch;

  const int kw0 = k0 + wave * 32;
  const int krow = kw0 + l32;
  const bool kvalid = krow < seg.len;
  // Fields used inside the lambdas below, as plain values (capturing the
  // kernel argument itself would make the compiler spill it to scratch).
  const uint16_t* const qbase = a.q;
  const uint16_t* const dobase = a.dout;
  const float* const lsebase = a.lse;
  const float* const delbase = a.delta;
  const bool causal = a.causal != 0;
  const int group = L.group;
  const int64_t q_head = L.q_head, q_row = L.q_row, r_head = L.r_head;
  const int len = seg.len;

  // K and V rows of this lane's key as B operands of S = Q K^T, dP = dO V^T.
  u32x4 kreg[D / 16], vreg[D / 16];
  {
    const rsrc_t rk = rows_rsrc(a.k + kvoff, kw0, seg.len, L.kv_row);
    const rsrc_t rv = rows_rsrc(a.v + kvoff, kw0, seg.len, L.kv_row);
    const int base = l32 * (int)(L.kv_row * 2) + 16 * half;
#pragma unroll
    for (int c = 0; c < D / 16; ++c) {
      kreg[c] = bload16(rk, base + 32 * c);
      vreg[c] = bload16(rv, base + 32 * c);
    }
  }

  f32x16 dkacc[D / 32], dvacc[D / 32];
#pragma unroll
  for (int db = 0; db < D / 32; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      dkacc[db][r] = 0.f;
      dvacc[db][r] = 0.f;
    }

  // Iterations run over (group head g, query tile it) with it from the first
  // tile that can see key k0.
  const int it0 = a.causal ? k0 / kTileRows : 0;
  const int nqt = (seg.len + kTileRows - 1) / kTileRows;
  const int per_head = nqt - it0;
  const int niter = per_head * L.group;

  const Tile dma(wave, lane, (int)(L.q_row * 2));
  const RowReader<D> rr(l32, half);
  const TransReader<D> trr(lane);
  const float sl2 = a.scale_log2;

  auto issue = [&](int n, uint16_t* q, uint16_t* dout, float* lse, float* del) __attribute__((always_inline)) {
    const int g = n / per_head;
    const int qb = (it0 + n % per_head) * kTileRows;
    const int h = hk * group + g;
    const int64_t qoff = qseg + (int64_t)h * q_head;
    dma.load(rows_rsrc(qbase + qoff, qb, len, q_row), q, wave);
    dma.load(rows_rsrc(dobase + qoff, qb, len, q_row), dout, wave);
    const int64_t r = rseg + (int64_t)h * r_head;
    if (wave == 0) {
      load_rowvec(lsebase + r, qb, len, lse, lane);
      load_rowvec(delbase + r, qb, len, del, lane);
    }
  };

  auto compute = [&](int n, const uint16_t* q, const uint16_t* dout, const float* lse,
                     const float* del) __attribute__((always_inline)) {
    const int qb = (it0 + n % per_head) * kTileRows;
#pragma unroll
    for (int sb = 0; sb < 2; ++sb) {
      f32x16 s, dp;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        s[r] = 0.f;
        dp[r] = 0.f;
      }
#pragma unroll
      for (int c = 0; c < D / 16; ++c) {
        const int o = rr.rm[c] + 32 * sb * D;
        s = mfma32(ld16(q + o), kreg[c], s);
        dp = mfma32(ld16(dout + o), vreg[c], dp);
      }
      // s[r], dp[r]: query qb + 32sb + 8(r/4) + 4half + r%4, key krow.
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const f32x4 l4 = *reinterpret_cast<const f32x4*>(&lse[32 * sb + 8 * g + 4 * half]);
#pragma unroll
        for (int i = 0; i < 4; ++i)
          s[4 * g + i] = fast_exp2(__builtin_fmaf(s[4 * g + i], sl2, -l4[i] * kLog2e));
      }
      if (causal && qb + 32 * sb < kw0 + 31) {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int q = qb + 32 * sb + 8 * (r / 4) + 4 * half + (r % 4);
          s[r] = krow > q ? 0.f : s[r];
        }
      }
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const f32x4 d4 = *reinterpret_cast<const f32x4*>(&del[32 * sb + 8 * g + 4 * half]);
#pragma unroll
        for (int i = 0; i < 4; ++i) dp[4 * g + i] = s[4 * g + i] * (dp[4 * g + i] - d4[i]);   // dS
      }
      // dV^T[d][key] += sum_q dO^T[d][q] P[q][key];  dK^T += Q^T dS; the A
      // operands are read transposed out of the row-major dO and Q tiles.
#pragma unroll
      for (int c = 0; c < 2; ++c) {
        const u32x4 pb = pack_chunk(s, c);
        const u32x4 dsb = pack_chunk(dp, c);
        const int rc = 16 * (2 * sb + c) * D;
#pragma unroll
        for (int db = 0; db < D / 32; ++db) {
          const u32x2 dlo = ld_tr(dout + trr.tr[db][0] + rc), dhi = ld_tr(dout + trr.tr[db][1] + rc);
          dvacc[db] = mfma32(u32x4{dlo[0], dlo[1], dhi[0], dhi[1]}, pb, dvacc[db]);
          const u32x2 qlo = ld_tr(q + trr.tr[db][0] + rc), qhi = ld_tr(q + trr.tr[db][1] + rc);
          dkacc[db] = mfma32(u32x4{qlo[0], qlo[1], qhi[0], qhi[1]}, dsb, dkacc[db]);
        }
      }
    }
  };

  auto step0 = [&](int n) __attribute__((always_inline)) {   // compute from stage 0, prefetch into stage 1
    wait_vm<0>();
    __syncthreads();
    if (n + 1 < niter) issue(n + 1, sq1, sdo1, sl1, sd1);
    compute(n, sq0, sdo0, sl0, sd0);
  };
  auto step1 = [&](int n) __attribute__((always_inline)) {   // compute from stage 1, prefetch into stage 0
    wait_vm<0>();
    __syncthreads();
    if (n + 1 < niter) issue(n + 1, sq0, sdo0, sl0, sd0);
    compute(n, sq1, sdo1, sl1, sd1);
  };

  if (niter > 0) issue(0, sq0, sdo0, sl0, sd0);
  wait_vm<0>();
  int n = 0;
  for (; n + 1 < niter; n += 2) {
    step0(n);
    step1(n + 1);
  }
  if (n < niter) step0(n);

  if (kvalid) {
    const int64_t off = kvoff + (int64_t)krow * L.kv_row;
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        u32x2 wk, wv;
        wk[0] = pack_bf16(dkacc[db][4 * g + 0] * a.scale, dkacc[db][4 * g + 1] * a.scale);
        wk[1] = pack_bf16(dkacc[db][4 * g + 2] * a.scale, dkacc[db][4 * g + 3] * a.scale);
        wv[0] = pack_bf16(dvacc[db][4 * g + 0], dvacc[db][4 * g + 1]);
        wv[1] = pack_bf16(dvacc[db][4 * g + 2], dvacc[db][4 * g + 3]);
        st8(a.dk + off + 32 * db + 8 * g + 4 * half, wk);
        st8(a.dv + off + 32 * db + 8 * g + 4 * half, wv);
      }
  }
}

// Explicit instantiations: without them the host compiler may skip the
// launch stubs of these templates (leaving undefined symbols in the library).
template __global__ void bwd_dq_kernel<64>(BwdArgs);
template __global__ void bwd_dq_kernel<128>(BwdArgs);
template __global__ void bwd_dkdv_kernel<64>(BwdArgs);
template __global__ void bwd_dkdv_kernel<128>(BwdArgs);

}  // namespace

hipError_t launch_bwd(const BwdArgs& a, int D, int phases, hipStream_t stream) {
  const dim3 gq((unsigned)(a.L.nseg * a.L.Hq), (unsigned)((a.L.S + kQM - 1) / kQM));
  const dim3 gk((unsigned)(a.L.nseg * a.L.Hkv), (unsigned)((a.L.S + kKN - 1) / kKN));
  if (phases & 1) {
    if (D == 64)
      hipLaunchKernelGGL(bwd_dq_kernel<64>, gq, dim3(kThreads), 0, stream, a);
    else
      hipLaunchKernelGGL(bwd_dq_kernel<128>, gq, dim3(kThreads), 0, stream, a);
  }
  if (phases & 2) {
    if (D == 64)
      hipLaunchKernelGGL(bwd_dkdv_kernel<64>, gk, dim3(kThreads), 0, stream, a);
    else
      hipLaunchKernelGGL(bwd_dkdv_kernel<128>, gk, dim3(kThreads), 0, stream, a);
  }
  return hipGetLastError();
}

}  // namespace attn
