// Fused attention forward for gfx950: O = softmax(scale Q K^T + mask) V and
// the row log-sum-exp, with the online-softmax recurrence of the corrected
// FlashAttention-3 Algorithm 2 (PTXBench, Appendix A): per query block keep
// the running row maximum m and row sum l, rescale the output accumulator by
// exp(m_old - m_new) whenever the maximum moves, and normalise by l in the
// epilogue, where L = m + log l.
//
// Work split: one workgroup of 4 wavefronts per (segment, query head, 128
// query rows); each wavefront owns 32 query rows.  The wavefront computes the
// transposed score tile S^T = K Q^T on MFMA, so lane l holds every score of
// query (l % 32) against half of the tile's keys: the row maximum and row sum
// are in-lane reductions plus one exchange with lane l ^ 32.  P^T, rounded to
// bf16, is then already laid out as the B operand of O^T += V^T P^T.
//
// K tiles are stored row-major in LDS (each lane reads 16 contiguous bytes of
// one key row); V tiles are transposed on their way into LDS so that the A
// operand V^T is read as two 8-byte pieces.  The next tile's global loads are
// issued before the current tile's MFMAs and land in LDS after them.
#include "attn_kernels.hpp"
#include "device_common.hpp"

namespace attn {
namespace {

constexpr int kThreads = 256;
constexpr int kBM = 128;   // query rows per workgroup
constexpr int kBN = 64;    // keys per iteration

template <int D>
struct FwdTile {
  static constexpr int KS = D + 8;                  // K row stride, bf16 (16 B pad)
  static constexpr int VS = kBN + 4;                // V^T row stride, bf16 (8 B pad)
  static constexpr int CPR = D / 8;                 // 16-byte chunks per row
  static constexpr int KPASS = kBN * CPR / kThreads;
  static constexpr int KROWS = kThreads / CPR;      // K rows per pass
  static constexpr int VBLK = (kBN / 4) * CPR;      // 4-key x 8-d blocks of V
  static_assert(KPASS * KROWS == kBN, "K tile split");
  static_assert(VBLK <= kThreads, "V tile split");
};

template <int D>
__global__ __launch_bounds__(kThreads, 2) void fwd_kernel(FwdArgs a) {
  using T = FwdTile<D>;
  __shared__ __attribute__((aligned(16))) uint16_t sk[kBN * T::KS];
  __shared__ __attribute__((aligned(16))) uint16_t svt[D * T::VS];

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int l32 = lane & 31, half = lane >> 5;

  const Layout& L = a.L;
  const int z = blockIdx.x / L.Hq, h = blockIdx.x % L.Hq;
  const int hk = h / L.group;
  const Segment seg = segment_of(L, z);
  const int qt = (int)gridDim.y - 1 - (int)blockIdx.y;  // longest rows first
  const int q0 = qt * kBM;
  if (q0 >= seg.len) return;

  const int64_t qoff = (L.cu ? (int64_t)seg.start * L.q_row : (int64_t)z * L.q_batch) +
                       (int64_t)h * L.q_head;
  const int64_t kvoff = (L.cu ? (int64_t)seg.start * L.kv_row : (int64_t)z * L.kv_batch) +
                        (int64_t)hk * L.kv_head;
  const int64_t roff = (L.cu ? (int64_t)seg.start : (int64_t)z * L.r_batch) +
                       (int64_t)h * L.r_head;
  const uint16_t* kp = a.k + kvoff;
  const uint16_t* vp = a.v + kvoff;

  // This lane's query row, held as B operands of S^T = K Q^T:
  // qreg[c] = Q[qrow][16c + 8*half .. +8].
  const int qw0 = q0 + wave * 32;
  const int qrow = qw0 + l32;
  u32x4 qreg[D / 16];
#pragma unroll
  for (int c = 0; c < D / 16; ++c)
    qreg[c] = qrow < seg.len ? ld16(a.q + qoff + (int64_t)qrow * L.q_row + 16 * c + 8 * half)
                             : u32x4{0u, 0u, 0u, 0u};

  const int kend = a.causal ? min(seg.len, q0 + kBM) : seg.len;
  const int nkt = (kend + kBN - 1) / kBN;

  // Staging registers for the next K / V tile.
  u32x4 kst[T::KPASS];
  u32x4 vst[4];
  const int krow_ld = tid / T::CPR, kch = tid % T::CPR;   // K: row, chunk
  const int vkg = tid / T::CPR, vdc = tid % T::CPR;       // V: key group, d chunk
  auto gload = [&](int kt) {
    const int k0 = kt * kBN;
#pragma unroll
    for (int p = 0; p < T::KPASS; ++p) {
      const int key = k0 + p * T::KROWS + krow_ld;
      kst[p] = key < seg.len ? ld16(kp + (int64_t)key * L.kv_row + 8 * kch) : u32x4{0u, 0u, 0u, 0u};
    }
    if (tid < T::VBLK) {
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const int key = k0 + 4 * vkg + i;
        vst[i] = key < seg.len ? ld16(vp + (int64_t)key * L.kv_row + 8 * vdc) : u32x4{0u, 0u, 0u, 0u};
      }
    }
  };
  auto sstore = [&]() {
#pragma unroll
    for (int p = 0; p < T::KPASS; ++p) st16(&sk[(p * T::KROWS + krow_ld) * T::KS + 8 * kch], kst[p]);
    if (tid < T::VBLK) {
      u32x2 cols[8];
      transpose4x8(vst, cols);
#pragma unroll
      for (int e = 0; e < 8; ++e) st8(&svt[(8 * vdc + e) * T::VS + 4 * vkg], cols[e]);
    }
  };

  f32x16 oacc[D / 32];
#pragma unroll
  for (int db = 0; db < D / 32; ++db)
#pragma unroll
    for (int r = 0; r < 16; ++r) oacc[db][r] = 0.f;
  float m = -INFINITY;   // running max of scale*log2(e)*s for query qrow
  float lsum = 0.f;      // this lane's share of the running row sum

  gload(0);
  sstore();
  __syncthreads();
  for (int kt = 0; kt < nkt; ++kt) {
    if (kt + 1 < nkt) gload(kt + 1);
    const int k0 = kt * kBN;
    // A tile whose first key is after this wavefront's last query is fully
    // masked for it and changes nothing.
    if (!a.causal || k0 <= qw0 + 31) {
      f32x16 s[2];
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) s[kb][r] = 0.f;
#pragma unroll
      for (int c = 0; c < D / 16; ++c)
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
          s[kb] = mfma32(ld16(&sk[(32 * kb + l32) * T::KS + 16 * c + 8 * half]), qreg[c], s[kb]);

      // s[kb][r] is the score of key k0 + 32kb + 8(r/4) + 4half + r%4.
      const bool need_mask = (a.causal && k0 + kBN - 1 > qw0) || (k0 + kBN > seg.len);
      float mx = -INFINITY;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          float t = s[kb][r] * a.scale_log2;
          if (need_mask) {
            const int key = k0 + 32 * kb + 8 * (r / 4) + 4 * half + (r % 4);
            if ((a.causal && key > qrow) || key >= seg.len) t = -INFINITY;
          }
          s[kb][r] = t;
          mx = fmaxf(mx, t);
        }
      mx = fmaxf(mx, swap_halves(mx));
      const float mnew = fmaxf(m, mx);
      const float mref = mnew == -INFINITY ? 0.f : mnew;
      const float alpha = fast_exp2(m - mref);
      float rs = 0.f;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float p = fast_exp2(s[kb][r] - mref);
          s[kb][r] = p;
          rs += p;
        }
      lsum = lsum * alpha + rs;
      m = mnew;
#pragma unroll
      for (int db = 0; db < D / 32; ++db)
#pragma unroll
        for (int r = 0; r < 16; ++r) oacc[db][r] *= alpha;

      // O^T[d][q] += sum_key V^T[d][key] P^T[key][q]; chunk c = keys 16c..16c+15.
      u32x4 pb[4];
#pragma unroll
      for (int c = 0; c < 4; ++c) pb[c] = pack_chunk(s[c >> 1], c & 1);
#pragma unroll
      for (int db = 0; db < D / 32; ++db)
#pragma unroll
        for (int c = 0; c < 4; ++c) {
          const uint16_t* row = &svt[(32 * db + l32) * T::VS + 16 * c + 4 * half];
          const u32x2 lo = ld8(row), hi = ld8(row + 8);
          oacc[db] = mfma32(u32x4{lo[0], lo[1], hi[0], hi[1]}, pb[c], oacc[db]);
        }
    }
    __syncthreads();
    if (kt + 1 < nkt) {
      sstore();
      __syncthreads();
    }
  }

  // Epilogue: O = O / l, L = (m + log2 l) ln 2.
  lsum += swap_halves(lsum);
  if (qrow < seg.len) {
    const float inv = lsum > 0.f ? 1.f / lsum : 0.f;
    uint16_t* op = a.o + qoff + (int64_t)qrow * L.q_row;
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        u32x2 w;
        w[0] = pack_bf16(oacc[db][4 * g + 0] * inv, oacc[db][4 * g + 1] * inv);
        w[1] = pack_bf16(oacc[db][4 * g + 2] * inv, oacc[db][4 * g + 3] * inv);
        st8(op + 32 * db + 8 * g + 4 * half, w);
      }
    if (half == 0) a.lse[roff + qrow] = lsum > 0.f ? (m + log2f(lsum)) * kLn2 : -INFINITY;
  }
}

}  // namespace

hipError_t launch_fwd(const FwdArgs& a, int D, hipStream_t stream) {
  const dim3 grid((unsigned)(a.L.nseg * a.L.Hq), (unsigned)((a.L.S + kBM - 1) / kBM));
  if (D == 64)
    hipLaunchKernelGGL(fwd_kernel<64>, grid, dim3(kThreads), 0, stream, a);
  else
    hipLaunchKernelGGL(fwd_kernel<128>, grid, dim3(kThreads), 0, stream, a);
  return hipGetLastError();
}

}  // namespace attn
