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
// Operand layouts follow device_common.hpp: accumulator tiles are fed back
// as B operands directly; operands whose reduction index runs along rows in
// memory (K^T, Q^T, dO^T) are transposed on their way into LDS.
#include "attn_kernels.hpp"
#include "device_common.hpp"

namespace attn {
namespace {

constexpr int kThreads = 256;

// Read offsets of this lane into a swizzled row-major [64][D] LDS tile for an
// MFMA operand over rows 32*b + (lane % 32): element offset of the 16-byte
// chunk 2c + half.  The swizzle does not depend on row bit 5, so the two
// 32-row blocks differ by a constant.
template <int D>
struct RowTileReader {
  int off[D / 16];
  __device__ __forceinline__ RowTileReader(int l32, int half) {
    const int x = swz_row<D>(l32);
#pragma unroll
    for (int c = 0; c < D / 16; ++c) off[c] = l32 * D + 8 * ((2 * c + half) ^ x);
  }
  __device__ __forceinline__ int at(int b, int c) const { return off[c] + 32 * b * D; }
};

// Store a 4-row x 8-column block (rows 4*rg .. 4*rg+3, column chunk cc) into
// a swizzled row-major [64][D] tile and, optionally, a transposed [D][kTS]
// tile.
template <int D>
__device__ __forceinline__ void store_block(uint16_t* rowtile, uint16_t* ttile, const BlockMap<D>& m,
                                            const u32x4 (&blk)[4]) {
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int j = store_row_order<D>(i, m.cc);
    const int r = 4 * m.rg + j;
    st16(&rowtile[r * D + 8 * (m.cc ^ swz_row<D>(r))], blk[j]);
  }
  if (ttile) {
    u32x2 cols[8];
    transpose4x8(blk, cols);
#pragma unroll
    for (int e = 0; e < 8; ++e) st8(&ttile[(8 * m.cc + e) * kTS + 4 * m.rg], cols[e]);
  }
}

// ---------------------------------------------------------------------------
// dQ (and Delta)
// ---------------------------------------------------------------------------
constexpr int kQM = 128;   // query rows per workgroup
constexpr int kQN = 64;    // keys per iteration

template <int D>
__global__ __launch_bounds__(kThreads, 1) void bwd_dq_kernel(BwdArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t sk[kQN * D];
  __shared__ __attribute__((aligned(16))) uint16_t skt[D * kTS];
  __shared__ __attribute__((aligned(16))) uint16_t sv[kQN * D];

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = wave_id();
  const int l32 = lane & 31, half = lane >> 5;

  const Layout& L = a.L;
  const int z = blockIdx.x / L.Hq, h = blockIdx.x % L.Hq;
  const int hk = h / L.group;
  const Segment seg = segment_of(L, z);
  const int qt = (int)gridDim.y - 1 - (int)blockIdx.y;
  const int q0 = qt * kQM;
  if (q0 >= seg.len) return;

  const int64_t qoff = (L.cu ? (int64_t)seg.start * L.q_row : (int64_t)z * L.q_batch) +
                       (int64_t)h * L.q_head;
  const int64_t kvoff = (L.cu ? (int64_t)seg.start * L.kv_row : (int64_t)z * L.kv_batch) +
                        (int64_t)hk * L.kv_head;
  const int64_t roff = (L.cu ? (int64_t)seg.start : (int64_t)z * L.r_batch) +
                       (int64_t)h * L.r_head;
  const uint16_t* kp = a.k + kvoff;
  const uint16_t* vp = a.v + kvoff;
  const int kvrow_b = (int)(L.kv_row * 2);

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
  float lse2 = INFINITY;   // exp2(s*scale*log2e - lse2) = 0 for rows outside
  if (valid) {
    const float l = a.lse[roff + qrow];
    lse2 = l == -INFINITY ? INFINITY : l * kLog2e;
    if (half == 0) a.delta[roff + qrow] = delta;
  }

  const int kend = a.causal ? min(seg.len, q0 + kQM) : seg.len;
  const int nkt = (kend + kQN - 1) / kQN;

  // Staging: K and V as 4-row x 8-column blocks.
  const BlockMap<D> bm(tid);
  u32x4 kst[4], vst[4];
  auto gload = [&](int kt) {
    if (!bm.active) return;
    const int k0 = kt * kQN;
    const rsrc_t rk = rows_rsrc(kp, k0, seg.len, L.kv_row);
    const rsrc_t rv = rows_rsrc(vp, k0, seg.len, L.kv_row);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int off = (4 * bm.rg + i) * kvrow_b + 16 * bm.cc;
      kst[i] = bload16(rk, off);
      vst[i] = bload16(rv, off);
    }
  };
  auto sstore = [&]() {
    if (!bm.active) return;
    store_block<D>(sk, skt, bm, kst);
    store_block<D>(sv, nullptr, bm, vst);
  };

  const RowTileReader<D> rd(l32, half);
  const uint16_t* ktrd = &skt[l32 * kTS + 4 * half];

  f32x16 dqacc[D / 32];
#pragma unroll
  for (int db = 0; db < D / 32; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) dqacc[db][r] = 0.f;
  const float sl2 = a.scale_log2;

  gload(0);
  sstore();
  __syncthreads();
  for (int kt = 0; kt < nkt; ++kt) {
    if (kt + 1 < nkt) gload(kt + 1);
    const int k0 = kt * kQN;
    if (!a.causal || k0 <= qw0 + 31) {
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
          const int o = rd.at(kb, c);
          s[kb] = mfma32(ld16(&sk[o]), qreg[c], s[kb]);
          dp[kb] = mfma32(ld16(&sv[o]), doreg[c], dp[kb]);
        }
      const bool need_mask = (a.causal && k0 + kQN - 1 > qw0) || (k0 + kQN > seg.len);
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          float p = fast_exp2(__builtin_fmaf(s[kb][r], sl2, -lse2));
          if (need_mask) {
            const int key = k0 + 32 * kb + 8 * (r / 4) + 4 * half + (r % 4);
            p = ((a.causal && key > qrow) || key >= seg.len) ? 0.f : p;
          }
          s[kb][r] = p * (dp[kb][r] - delta);   // dS^T
        }
      // dQ^T[d][q] += sum_key K^T[d][key] dS^T[key][q]
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        const u32x4 b = pack_chunk(s[c >> 1], c & 1);
#pragma unroll
        for (int db = 0; db < D / 32; ++db) {
          const uint16_t* row = ktrd + 32 * db * kTS + 16 * c;
          const u32x2 lo = ld8(row), hi = ld8(row + 8);
          dqacc[db] = mfma32(u32x4{lo[0], lo[1], hi[0], hi[1]}, b, dqacc[db]);
        }
      }
    }
    __syncthreads();
    if (kt + 1 < nkt) {
      sstore();
      __syncthreads();
    }
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
constexpr int kKM = 64;    // query rows per iteration

template <int D>
__global__ __launch_bounds__(kThreads, 1) void bwd_dkdv_kernel(BwdArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t sq[kKM * D];
  __shared__ __attribute__((aligned(16))) uint16_t sqt[D * kTS];
  __shared__ __attribute__((aligned(16))) uint16_t sdo[kKM * D];
  __shared__ __attribute__((aligned(16))) uint16_t sdot[D * kTS];
  __shared__ __attribute__((aligned(16))) float slse[kKM];
  __shared__ __attribute__((aligned(16))) float sdelta[kKM];

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = wave_id();
  const int l32 = lane & 31, half = lane >> 5;

  const Layout& L = a.L;
  const int z = blockIdx.x / L.Hkv, hk = blockIdx.x % L.Hkv;
  const Segment seg = segment_of(L, z);
  const int k0 = (int)blockIdx.y * kKN;   // lowest keys (most work) first
  if (k0 >= seg.len) return;

  const int64_t kvoff = (L.cu ? (int64_t)seg.start * L.kv_row : (int64_t)z * L.kv_batch) +
                        (int64_t)hk * L.kv_head;
  const int64_t qseg = L.cu ? (int64_t)seg.start * L.q_row : (int64_t)z * L.q_batch;
  const int64_t rseg = L.cu ? (int64_t)seg.start : (int64_t)z * L.r_batch;
  const int qrow_b = (int)(L.q_row * 2);

  const int kw0 = k0 + wave * 32;
  const int krow = kw0 + l32;
  const bool kvalid = krow < seg.len;

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
  const int it0 = a.causal ? k0 / kKM : 0;
  const int nqt = (seg.len + kKM - 1) / kKM;
  const int per_head = nqt - it0;
  const int niter = per_head * L.group;

  const BlockMap<D> bm(tid);
  u32x4 qst[4], dost[4];
  float lst = INFINITY, dst = 0.f;
  auto gload = [&](int n) {
    const int g = n / per_head;
    const int qb = (it0 + n % per_head) * kKM;
    const int h = hk * L.group + g;
    const int64_t qoff = qseg + (int64_t)h * L.q_head;
    if (bm.active) {
      const rsrc_t rq = rows_rsrc(a.q + qoff, qb, seg.len, L.q_row);
      const rsrc_t rdo = rows_rsrc(a.dout + qoff, qb, seg.len, L.q_row);
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int off = (4 * bm.rg + i) * qrow_b + 16 * bm.cc;
        qst[i] = bload16(rq, off);
        dost[i] = bload16(rdo, off);
      }
    }
    if (tid < kKM) {
      const int q = qb + tid;
      const int64_t r = rseg + (int64_t)h * L.r_head + q;
      if (q < seg.len) {
        const float l = a.lse[r];
        lst = l == -INFINITY ? INFINITY : l * kLog2e;
        dst = a.delta[r];
      } else {
        lst = INFINITY;   // rows past the end contribute nothing
        dst = 0.f;
      }
    }
  };
  auto sstore = [&]() {
    if (bm.active) {
      store_block<D>(sq, sqt, bm, qst);
      store_block<D>(sdo, sdot, bm, dost);
    }
    if (tid < kKM) {
      slse[tid] = lst;
      sdelta[tid] = dst;
    }
  };

  const RowTileReader<D> rd(l32, half);
  const int trd = l32 * kTS + 4 * half;
  const float sl2 = a.scale_log2;

  if (niter > 0) {
    gload(0);
    sstore();
  }
  __syncthreads();
  for (int n = 0; n < niter; ++n) {
    if (n + 1 < niter) gload(n + 1);
    const int qb = (it0 + n % per_head) * kKM;
#pragma unroll
    for (int sb = 0; sb < kKM / 32; ++sb) {
      const int qs0 = qb + 32 * sb;
      // Skip sub-blocks whose every query precedes every key of this wave.
      if (a.causal && qs0 + 31 < kw0) continue;
      f32x16 s, dp;
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        s[r] = 0.f;
        dp[r] = 0.f;
      }
#pragma unroll
      for (int c = 0; c < D / 16; ++c) {
        const int o = rd.at(sb, c);
        s = mfma32(ld16(&sq[o]), kreg[c], s);
        dp = mfma32(ld16(&sdo[o]), vreg[c], dp);
      }
      // s[r], dp[r]: query qs0 + 8(r/4) + 4half + r%4, key krow.
      const bool need_mask = a.causal && qs0 < kw0 + 31;
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const f32x4 l4 = *reinterpret_cast<const f32x4*>(&slse[32 * sb + 8 * g + 4 * half]);
        const f32x4 d4 = *reinterpret_cast<const f32x4*>(&sdelta[32 * sb + 8 * g + 4 * half]);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const int r = 4 * g + i;
          float p = fast_exp2(__builtin_fmaf(s[r], sl2, -l4[i]));
          if (need_mask) p = krow > qs0 + 8 * g + 4 * half + i ? 0.f : p;
          s[r] = p;
          dp[r] = p * (dp[r] - d4[i]);   // dS
        }
      }
      // dV^T[d][key] += sum_q dO^T[d][q] P[q][key];  dK^T += Q^T dS.
#pragma unroll
      for (int c = 0; c < 2; ++c) {
        const u32x4 pb = pack_chunk(s, c);
        const u32x4 dsb = pack_chunk(dp, c);
#pragma unroll
        for (int db = 0; db < D / 32; ++db) {
          const int ro = trd + 32 * db * kTS + 32 * sb + 16 * c;
          const u32x2 dlo = ld8(&sdot[ro]), dhi = ld8(&sdot[ro + 8]);
          dvacc[db] = mfma32(u32x4{dlo[0], dlo[1], dhi[0], dhi[1]}, pb, dvacc[db]);
          const u32x2 qlo = ld8(&sqt[ro]), qhi = ld8(&sqt[ro + 8]);
          dkacc[db] = mfma32(u32x4{qlo[0], qlo[1], qhi[0], qhi[1]}, dsb, dkacc[db]);
        }
      }
    }
    __syncthreads();
    if (n + 1 < niter) {
      sstore();
      __syncthreads();
    }
  }

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
