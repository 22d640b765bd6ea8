// Fused attention forward for gfx950: O = softmax(scale Q K^T + mask) V and
// the row log-sum-exp, with the online-softmax recurrence of the corrected
// FlashAttention-3 Algorithm 2 (PTXBench, Appendix A): per query block keep
// a running row maximum m and row sum l, rescale the output accumulator by
// exp(m_old - m_new) when the maximum moves, and normalise by l in the
// epilogue, where L = m + log l.
//
// Work split: one workgroup of 4 wavefronts per (segment, query head,
// 128-row query block), the blocks with the most key tiles first, two
// workgroups per CU; each wavefront owns 32 query rows.  A paged prefill
// whose grid leaves CUs idle instead runs 8 wavefronts per block, one
// workgroup per CU: the two halves of the workgroup take alternate key
// tiles of the same rows, and the upper half hands its softmax state and
// output to the lower through LDS at the end, which halves the longest
// walk over keys without writing partial results to memory.  The wavefront computes the transposed score tile S^T = K Q^T on
// MFMA, so lane l holds every score of query (l % 32) against half of the
// tile's keys: the row maximum and row sum are in-lane reductions plus one
// exchange with lane l ^ 32.  P^T, rounded to bf16, is then already laid out
// as the B operand of O^T += V^T P^T.
//
// The reference maximum used for P is only moved when a tile's row maximum
// exceeds it by more than 2^8 (in exp2 units), so most tiles skip the
// rescale of O and l.  This is exact: O and l always share one reference,
// and entries of P stay below 2^8, far inside fp32 and bf16 range.
//
// K and V tiles go from global memory straight into a ring of LDS stages
// (buffer_load ... lds, bounded at the sequence end so that rows past it read
// as zero), issued a stage ahead, with one barrier per tile.  With a paged
// cache (page size 1) each lane's copy offset comes from the page number of
// its tile row, so the gather costs no extra pass; the page numbers are
// fetched one tile ahead, and a page outside the cache reads as zeros.  Both stay
// row-major in LDS: K is read as 16-byte rows, and the A operand V^T comes
// out of the V tile through the transposing read ds_read_b64_tr_b16, so no
// register staging or transposing store is needed.
#include "attn_kernels.hpp"
#include "device_common.hpp"

namespace attn {
namespace {

constexpr int kThreads = 256;
constexpr int kBM = kFwdBlockRows;   // query rows per workgroup
static_assert(kFwdSplitKeys % 128 == 0, "a chunk starts on an even key tile (stage 0)");
constexpr int kBN = 64;    // keys per iteration
constexpr float kRescaleSlack = 8.0f;   // log2 of the largest P entry allowed

// Two LDS stages (2 x 32 KiB at D = 128 and at D = 96, whose rows are padded
// to 128 elements; two workgroups per CU), declared as
// separate objects so that the compiler can tell a stage being filled by DMA
// from the one being read and does not wait for the prefetch.  With KS = 2
// key halves each stage holds two tiles (one per half; one workgroup per CU).

template <int D, bool PAGED, int KS>
__global__ __launch_bounds__(kThreads * KS, KS == 1 ? 2 : 1) void fwd_kernel(FwdArgs a) {
  static_assert(KS == 1 || (KS == 2 && PAGED), "key halves only in the paged prefill");
  using Tile = AsyncTile<D>;
  constexpr int P = Tile::P;   // LDS row pitch (elements)
  __shared__ __attribute__((aligned(1024))) uint16_t sk0[KS * Tile::ELEMS];
  __shared__ __attribute__((aligned(1024))) uint16_t sk1[KS * Tile::ELEMS];
  __shared__ __attribute__((aligned(1024))) uint16_t sv0[KS * Tile::ELEMS];
  __shared__ __attribute__((aligned(1024))) uint16_t sv1[KS * Tile::ELEMS];

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave_all = wave_id();
  // Row group (32 query rows) and key half of this wavefront: key tiles
  // kt_lo + KS i + kh, i = 0, 1, ...
  const int wave = KS == 1 ? wave_all : wave_all & 3;
  const int kh = KS == 1 ? 0 : wave_all >> 2;
  const int l32 = lane & 31, half = lane >> 5;

  const Layout L = a.L;
  int z, h, p;
  if constexpr (PAGED) {
    z = blockIdx.x / L.Hq;
    h = blockIdx.x % L.Hq;
    p = (int)blockIdx.y;
  } else {
    int gk, j;
    if (!xcd_decode((int)blockIdx.x, a.xo, gk, j, p)) return;
    z = gk / L.Hkv;
    h = (gk % L.Hkv) * L.group + j;
  }
  const int hk = h / L.group;
  const Segment seg = segment_of(L, z);
  // Keys: the segment's own rows, or (paged) its pages; the queries are the
  // last seg.len of the kv_len key positions, so query row i sits at key
  // position i + dpos.
  const Segment kseg = PAGED ? kv_segment_of(L, z) : seg;
  const int kv_len = PAGED ? min(kseg.len, a.max_kvlen) : kseg.len;
  const int dpos = PAGED ? kv_len - seg.len : 0;
  // Unsplit: query block nqt - 1 - p, so that the blocks with the most key
  // tiles under the causal mask start first.  Split: query block p, key
  // chunk blockIdx.z.
  const int nqt = (seg.len + kBM - 1) / kBM;
  const int split = PAGED ? a.split : 0;
  const int chunk = (int)blockIdx.z;
  if (p >= nqt) return;

  {
    const int qt = split ? p : nqt - 1 - p;
    const int q0 = qt * kBM;
    const int64_t qoff = (int64_t)seg.start * L.q_row + (int64_t)z * L.q_batch +
                         (int64_t)h * L.q_head;
    const int64_t kvoff = PAGED ? (int64_t)hk * L.kv_head
                                : (int64_t)seg.start * L.kv_row + (int64_t)z * L.kv_batch +
                                      (int64_t)hk * L.kv_head;
    const int64_t roff = (int64_t)seg.start + (int64_t)z * L.r_batch + (int64_t)h * L.r_head;
    const uint16_t* kp = a.k + kvoff;
    const uint16_t* vp = a.v + kvoff;

    // This lane's query row, held as B operands of S^T = K Q^T:
    // qreg[c] = Q[qrow][16c + 8*half .. +8].
    const int qw0 = q0 + wave * 32;
    const int qrow = qw0 + l32;
    u32x4 qreg[D / 16];
    {
      const rsrc_t rq = rows_rsrc(a.q + qoff, qw0, seg.len, L.q_row);
      const int base = l32 * (int)(L.q_row * 2) + 16 * half;
#pragma unroll
      for (int c = 0; c < D / 16; ++c) qreg[c] = bload16(rq, base + 32 * c);
    }

    const int kend = a.causal ? min(kv_len, max(0, q0 + kBM + dpos)) : kv_len;
    const int nkt = (kend + kBN - 1) / kBN;
    // This workgroup's key tiles [kt_lo, kt_hi): all of them, or one chunk.
    // A block with no visible key has one (empty) chunk, which writes the
    // rows' O = 0 and L = -inf.
    const int nch = split && KS == 1 ? max(1, (kend + split - 1) / split) : 1;
    if (chunk >= nch) return;   // split only (unsplit grids have one z slice)
    const int kt_lo = nch > 1 ? chunk * (split / kBN) : 0;
    const int kt_hi = nch > 1 ? min(nkt, kt_lo + split / kBN) : nkt;

    const Tile dma(wave, lane, (int)(L.kv_row * 2));
    const RowReader<D> kr(l32, half);
    const TransReader<D> vr(lane);

    f32x16 oacc[D / 32];
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
      for (int r = 0; r < 16; ++r) oacc[db][r] = 0.f;
    float mref = -INFINITY;   // reference max of scale*log2(e)*s for query qrow
    float lsum = 0.f;         // this lane's share of the row sum, relative to mref
    // ... and of the sum of P rounded to bf16, the weights the PV products
    // actually use.  O is normalised by this sum, so that its weights add up
    // to one and the rounding of P largely cancels; L keeps the fp32 sum.
    float lq = 0.f;
    const bf16x2 ones = __builtin_bit_cast(bf16x2, 0x3f803f80u);
    const float sl2 = a.scale_log2;
    // Fields used inside the lambdas below, as plain values (capturing the
    // kernel argument itself can make the compiler spill it to scratch).
    const bool causal = a.causal != 0;
    // K/V rows are below 2^24 bytes (no wider than a q-like row, and 128
    // q-like rows are below 2^31 bytes, which the API checks).
    const int kv_rb = (int)(L.kv_row * 2);
    const int kv_cap = 0x7fffffff / kv_rb;

    // Paged keys: tile rows are gathered through the page indices, which are
    // fetched one tile ahead of the copies that use them.
    int pidx[Tile::NJ];
    const int num_pages = L.num_pages;
    const int cache_row_bytes = (int)(L.kv_row * 2);
    const int64_t cache_bytes = PAGED ? (int64_t)L.num_pages * L.kv_row * 2 - kvoff * 2 : 0;
    const rsrc_t kcache = make_rsrc(kp, cache_bytes);
    const rsrc_t vcache = make_rsrc(vp, cache_bytes);
    const rsrc_t ixr = make_rsrc(PAGED ? L.kv_idx + kseg.start : nullptr,
                                 PAGED ? (int64_t)kv_len * 4 : 0);
    auto fetch = [&](int kt) __attribute__((always_inline)) {
#pragma unroll
      for (int j = 0; j < Tile::NJ; ++j)
        pidx[j] = bload4(ixr, 4 * (kt * kBN + Tile::row_of(wave, j, lane)));
    };
    // Start the copies of tile kt into stages kd, vd (and, paged, the index
    // fetch of this half's next tile, kt + KS).
    auto load_tile = [&](int kt, uint16_t* kd, uint16_t* vd) __attribute__((always_inline)) {
      if constexpr (PAGED) {
        int off[Tile::NJ];
#pragma unroll
        for (int j = 0; j < Tile::NJ; ++j) {
          const int key = kt * kBN + Tile::row_of(wave, j, lane);
          off[j] = Tile::gather_off(wave, j, lane, pidx[j], key < kv_len, num_pages,
                                    cache_row_bytes);
        }
        dma.load_at(kcache, off, kd, wave);
        dma.load_at(vcache, off, vd, wave);
        if (kt + KS < kt_hi) fetch(kt + KS);
      } else {
        // kt < nkt, so the tile starts before kv_len.
        dma.load(rows_rsrc_rb(reinterpret_cast<const char*>(kp), kt * kBN, kv_len, kv_rb, kv_cap),
                 kd, wave);
        dma.load(rows_rsrc_rb(reinterpret_cast<const char*>(vp), kt * kBN, kv_len, kv_rb, kv_cap),
                 vd, wave);
      }
    };

    auto compute = [&](int kt, const uint16_t* kt_lds, const uint16_t* vt_lds) __attribute__((always_inline)) {
      const int k0 = kt * kBN;
      f32x16 s[2];
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) s[kb][r] = 0.f;
#pragma unroll
      for (int c = 0; c < D / 16; ++c)
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
          s[kb] = mfma32(ld16(kt_lds + kr.rm[c] + 32 * kb * P), qreg[c], s[kb]);
      // Keep the K operand reads several MFMAs ahead of their products (left
      // to itself, the scheduler issues them one or two ahead, so most of the
      // S products wait out an LDS read).
      {
        constexpr int NR = D / 8, LEAD = NR < 6 ? NR : 6;
        __builtin_amdgcn_sched_group_barrier(0x100, LEAD, 0);   // LDS reads
#pragma unroll
        for (int i = 0; i < NR - LEAD; ++i) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);    // MFMA
          __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        }
        __builtin_amdgcn_sched_group_barrier(0x008, LEAD, 0);
      }

      // s[kb][r] is the raw score of key k0 + 32kb + 8(r/4) + 4half + r%4.
      if ((a.causal && k0 + kBN - 1 > qw0 + dpos) || k0 + kBN > kv_len) {
#pragma unroll
        for (int kb = 0; kb < 2; ++kb)
#pragma unroll
          for (int r = 0; r < 16; ++r) {
            const int key = k0 + 32 * kb + 8 * (r / 4) + 4 * half + (r % 4);
            const bool masked = (a.causal && key > qrow + dpos) || key >= kv_len;
            s[kb][r] = masked ? -INFINITY : s[kb][r];
          }
      }
      float mx = s[0][0];
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[kb][r]);
      mx = max_halves(mx);
      const float mt = mx * sl2;   // this tile's row max in exp2 units
      if (__ballot(mt > mref + kRescaleSlack)) {
        const float mnew = fmaxf(mref, mt);
        // 0 on the first visible tile; 1 for a row that has seen no key yet
        // (both maxima -inf), whose O and l are still 0.
        const float alpha = mnew == -INFINITY ? 1.f : fast_exp2(mref - mnew);
        lsum *= alpha;
        lq *= alpha;
#pragma unroll
        for (int db = 0; db < D / 32; ++db)
#pragma unroll
          for (int r = 0; r < 16; ++r) oacc[db][r] *= alpha;
        mref = mnew;
      }
      const float mneg = mref == -INFINITY ? 0.f : -mref;
      float rs = 0.f;
#pragma unroll
      for (int kb = 0; kb < 2; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const float pe = fast_exp2(__builtin_fmaf(s[kb][r], sl2, mneg));
          s[kb][r] = pe;
          rs += pe;
        }
      lsum += rs;

      // O^T[d][q] += sum_key V^T[d][key] P^T[key][q]; chunk c = keys 16c..16c+15,
      // V^T read transposed out of the row-major V tile.
      float lq1 = 0.f;
#pragma unroll
      for (int c = 0; c < 4; ++c) {
        // P^T chunk c as bf16 pairs; each pair is also summed as rounded
        // (v_dot2 with (1, 1)) as soon as it is packed.
        u32x4 pb;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const uint32_t w = pack_bf16(s[c >> 1][8 * (c & 1) + 2 * j],
                                       s[c >> 1][8 * (c & 1) + 2 * j + 1]);
          pb[j] = w;
          if (j & 1)
            lq1 = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w), ones, lq1, false);
          else
            lq = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, w), ones, lq, false);
        }
#pragma unroll
        for (int db = 0; db < D / 32; ++db) {
          const u32x2 lo = ld_tr(vt_lds + vr.tr[db][0] + 16 * c * P);
          const u32x2 hi = ld_tr(vt_lds + vr.tr[db][1] + 16 * c * P);
          oacc[db] = mfma32(u32x4{lo[0], lo[1], hi[0], hi[1]}, pb, oacc[db]);
        }
      }
      lq += lq1;
    };
    // Step i (this half's tile kt_lo + KS i + kh, stage i % 2): wait for its
    // loads (this wavefront's, then everyone's through the barrier, which
    // also frees the stage read at step i - 1), start the loads of step
    // i + 1 into that stage, then compute.
    uint16_t* const k0s = sk0 + kh * Tile::ELEMS;
    uint16_t* const v0s = sv0 + kh * Tile::ELEMS;
    uint16_t* const k1s = sk1 + kh * Tile::ELEMS;
    uint16_t* const v1s = sv1 + kh * Tile::ELEMS;
    auto step = [&](int i, bool work, const uint16_t* kc, const uint16_t* vc, uint16_t* kn,
                    uint16_t* vn) __attribute__((always_inline)) {
      wait_vm<0>();
      __syncthreads();
      const int kt = kt_lo + KS * i + kh;
      if (kt + KS < kt_hi) load_tile(kt + KS, kn, vn);
      if (work) compute(kt, kc, vc);
    };

    // Tiles past this wavefront's last query are fully masked for it: the
    // wavefront only joins their barriers and loads.
    const int last_key = qw0 + 31 + dpos;   // the wavefront's last visible key (causal)
    const int nkt_w = causal ? (last_key < 0 ? 0 : min(kt_hi, last_key / kBN + 1)) : kt_hi;
    // Steps of the workgroup, and those in which this wavefront computes.
    const int nst = (kt_hi - kt_lo + KS - 1) / KS;
    const int nst_w = nkt_w > kt_lo + kh ? (nkt_w - kt_lo - kh + KS - 1) / KS : 0;
    if (kt_lo + kh < kt_hi) {
      if constexpr (PAGED) fetch(kt_lo + kh);
      load_tile(kt_lo + kh, k0s, v0s);
    }
    wait_vm<0>();   // Q rows and the first tile
    int i = 0;
    for (; i + 1 < nst_w; i += 2) {
      step(i, true, k0s, v0s, k1s, v1s);
      step(i + 1, true, k1s, v1s, k0s, v0s);
    }
    if (i < nst_w) {
      step(i, true, k0s, v0s, k1s, v1s);
      ++i;
    }
    for (; i < nst; ++i) {
      if (i & 1)
        step(i, false, k1s, v1s, k0s, v0s);
      else
        step(i, false, k0s, v0s, k1s, v1s);
    }

    // Epilogue: O = O / l, L = (m + log2 l) ln 2; or, for one chunk of
    // several, the chunk's O / l and m + log2 l (base 2) as a partial result.
    lsum = sum_halves(lsum);
    lq = sum_halves(lq);
    if constexpr (KS == 2) {
      // The upper half's state for the same rows and columns goes through
      // LDS (row group w uses stage object w, now free) to the lower half,
      // which rebases both onto the larger reference maximum and adds them.
      __syncthreads();   // every wavefront is done with the stages
      float* const xb = reinterpret_cast<float*>(wave == 0 ? sk0 : wave == 1 ? sk1
                                                 : wave == 2 ? sv0 : sv1);
      constexpr int NV = D / 2;   // output accumulator values per lane
      static_assert((NV + 3) * 64 * 4 <= KS * Tile::ELEMS * 2, "merge staging");
      if (kh == 1) {
#pragma unroll
        for (int db = 0; db < D / 32; ++db)
#pragma unroll
          for (int r = 0; r < 16; ++r) xb[(16 * db + r) * 64 + lane] = oacc[db][r];
        xb[NV * 64 + lane] = mref;
        xb[(NV + 1) * 64 + lane] = lsum;
        xb[(NV + 2) * 64 + lane] = lq;
      }
      __syncthreads();
      if (kh == 1) return;
      const float m1 = xb[NV * 64 + lane];
      const float mnew = fmaxf(mref, m1);
      // A half that saw no key has reference -inf and l = 0: weight 0.
      const float a0 = mref == -INFINITY ? 0.f : fast_exp2(mref - mnew);
      const float a1 = m1 == -INFINITY ? 0.f : fast_exp2(m1 - mnew);
      lsum = a0 * lsum + a1 * xb[(NV + 1) * 64 + lane];
      lq = a0 * lq + a1 * xb[(NV + 2) * 64 + lane];
      mref = mnew;
#pragma unroll
      for (int db = 0; db < D / 32; ++db)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          oacc[db][r] = a0 * oacc[db][r] + a1 * xb[(16 * db + r) * 64 + lane];
    }
    if (nch > 1) {
      if (qrow < seg.len) {
        const float inv = lq > 0.f ? 1.f / lq : 0.f;
        const int64_t slot = ((int64_t)(seg.start + qrow) * L.Hq + h) * a.nsplit + chunk;
        float* po = a.part_o + slot * D + 4 * half;
#pragma unroll
        for (int db = 0; db < D / 32; ++db)
#pragma unroll
          for (int g = 0; g < 4; ++g)
            *reinterpret_cast<f32x4*>(po + 32 * db + 8 * g) =
                f32x4{oacc[db][4 * g], oacc[db][4 * g + 1], oacc[db][4 * g + 2],
                      oacc[db][4 * g + 3]} *
                inv;
        if (half == 0) a.part_lse[slot] = lsum > 0.f ? mref + log2f(lsum) : -INFINITY;
      }
    } else if (qrow < seg.len) {
      const float inv = lq > 0.f ? 1.f / lq : 0.f;
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
      if (half == 0) a.lse[roff + qrow] = lsum > 0.f ? (mref + log2f(lsum)) * kLn2 : -INFINITY;
    }
  }
}

// Merge of a split paged prefill: for each query row of a block with more
// than one key chunk, O = sum_c 2^(L_c - M) O_c / sum_c 2^(L_c - M) and
// L = (M + log2 sum_c 2^(L_c - M)) ln 2, M = max_c L_c.  A chunk in which the
// row sees no key has L_c = -inf and weight 0; a row that sees no key at all
// gets O = 0 and L = -inf.  One workgroup of 4 wavefronts per (segment, query
// head, 32 rows of a query block); half a wavefront per row, 4 output columns
// per lane, kMergePasses rows per half wavefront.  Every load of the first
// kMergeU chunks of all its rows is issued before any is used: the chunk
// index is clamped into the row's chunks (the loads are always in bounds and
// need no branch) and the clamped repeats are dropped by selects.
constexpr int kMergePasses = 4;
constexpr int kMergeRows = 8 * kMergePasses;
constexpr int kMergeU = 4;

template <int D>
__global__ __launch_bounds__(256) void fwd_merge_kernel(FwdArgs a) {
  const int lane = threadIdx.x & 63, wave = wave_id();
  const Layout L = a.L;
  const int z = blockIdx.x / L.Hq, h = blockIdx.x % L.Hq;
  const Segment seg = segment_of(L, z);
  const int kv_len = min(kv_segment_of(L, z).len, a.max_kvlen);
  const int dpos = kv_len - seg.len;
  const int q0 = (int)blockIdx.y * kBM;
  if (q0 >= seg.len) return;
  const int kend = a.causal ? min(kv_len, max(0, q0 + kBM + dpos)) : kv_len;
  const int nch = (kend + a.split - 1) / a.split;
  if (nch <= 1) return;   // the forward wrote the block's rows itself
  const int row0 = q0 + (int)blockIdx.z * kMergeRows + 2 * wave + (lane >> 5);
  const int dl = 4 * (lane & 31);
  const bool col = dl < D;
  const int d = col ? dl : 0;

  float l[kMergePasses][kMergeU];
  f32x4 v[kMergePasses][kMergeU];
#pragma unroll
  for (int i = 0; i < kMergePasses; ++i) {
    const int row = min(row0 + 8 * i, seg.len - 1);
    const int64_t slot0 = ((int64_t)(seg.start + row) * L.Hq + h) * a.nsplit;
#pragma unroll
    for (int u = 0; u < kMergeU; ++u) {
      const int c = min(u, nch - 1);
      l[i][u] = a.part_lse[slot0 + c];
      v[i][u] = *reinterpret_cast<const f32x4*>(a.part_o + (slot0 + c) * D + d);
    }
  }
#pragma unroll
  for (int i = 0; i < kMergePasses; ++i) {
    const int row = row0 + 8 * i;
    if (row >= seg.len) break;
    const int64_t slot0 = ((int64_t)(seg.start + row) * L.Hq + h) * a.nsplit;
    const float* const pl = a.part_lse + slot0;
    const float* const po = a.part_o + slot0 * D + d;
    float M = -INFINITY;
#pragma unroll
    for (int u = 0; u < kMergeU; ++u)
      if (u < nch) M = fmaxf(M, l[i][u]);
    for (int c = kMergeU; c < nch; ++c) M = fmaxf(M, pl[c]);
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    float wsum = 0.f;
    if (M != -INFINITY) {
#pragma unroll
      for (int u = 0; u < kMergeU; ++u)
        if (u < nch) {
          const float w = fast_exp2(l[i][u] - M);
          wsum += w;
          acc += w * v[i][u];
        }
      for (int c = kMergeU; c < nch; ++c) {
        const float w = fast_exp2(pl[c] - M);
        wsum += w;
        acc += w * *reinterpret_cast<const f32x4*>(po + (int64_t)c * D);
      }
    }
    const float inv = wsum > 0.f ? 1.f / wsum : 0.f;
    if (col)
      st8(a.o + (int64_t)(seg.start + row) * L.q_row + (int64_t)h * L.q_head + d,
          u32x2{pack_bf16(acc[0] * inv, acc[1] * inv), pack_bf16(acc[2] * inv, acc[3] * inv)});
    if ((lane & 31) == 0)
      a.lse[(int64_t)seg.start + (int64_t)h * L.r_head + row] =
          wsum > 0.f ? (M + log2f(wsum)) * kLn2 : -INFINITY;
  }
}

template __global__ void fwd_merge_kernel<64>(FwdArgs);
template __global__ void fwd_merge_kernel<96>(FwdArgs);
template __global__ void fwd_merge_kernel<128>(FwdArgs);

// Explicit instantiations: without them the host compiler may skip the
// launch stubs of these templates (leaving undefined symbols in the library).
template __global__ void fwd_kernel<64, false, 1>(FwdArgs);
template __global__ void fwd_kernel<96, false, 1>(FwdArgs);
template __global__ void fwd_kernel<128, false, 1>(FwdArgs);
template __global__ void fwd_kernel<64, true, 1>(FwdArgs);
template __global__ void fwd_kernel<96, true, 1>(FwdArgs);
template __global__ void fwd_kernel<128, true, 1>(FwdArgs);
template __global__ void fwd_kernel<64, true, 2>(FwdArgs);
template __global__ void fwd_kernel<96, true, 2>(FwdArgs);
template __global__ void fwd_kernel<128, true, 2>(FwdArgs);

template <int D>
void launch_merge(const FwdArgs& a, dim3 grid, hipStream_t stream) {
  hipLaunchKernelGGL((fwd_merge_kernel<D>), grid, dim3(256), 0, stream, a);
}

template <bool PAGED, int KS = 1>
void launch_fwd_p(const FwdArgs& a, int D, dim3 grid, hipStream_t stream) {
  const dim3 block(kThreads * KS);
  if (D == 64)
    hipLaunchKernelGGL((fwd_kernel<64, PAGED, KS>), grid, block, 0, stream, a);
  else if (D == 96)
    hipLaunchKernelGGL((fwd_kernel<96, PAGED, KS>), grid, block, 0, stream, a);
  else
    hipLaunchKernelGGL((fwd_kernel<128, PAGED, KS>), grid, block, 0, stream, a);
}

}  // namespace

hipError_t launch_fwd(const FwdArgs& a, int D, hipStream_t stream) {
  const int nqt = (a.L.S + kBM - 1) / kBM;
  const unsigned heads = (unsigned)(a.L.nseg * a.L.Hq);
  if (a.L.kv_cu && a.split > 0) {
    // One workgroup per (query block, key chunk), then the merge.
    launch_fwd_p<true>(a, D, dim3(heads, (unsigned)nqt, (unsigned)a.nsplit), stream);
    const dim3 mg(heads, (unsigned)nqt, (unsigned)(kBM / kMergeRows));
    if (D == 64)
      launch_merge<64>(a, mg, stream);
    else if (D == 96)
      launch_merge<96>(a, mg, stream);
    else
      launch_merge<128>(a, mg, stream);
    return hipGetLastError();
  }
  // One workgroup per query block (see the kernel); unpaged launches in the
  // XCD-aware order.  A paged grid with fewer workgroups than CUs runs the
  // 8-wavefront form (key halves), one workgroup per CU.
  if (a.L.kv_cu) {
    if (paged_key_halves(heads, a.L.S))
      launch_fwd_p<true, 2>(a, D, dim3(heads, (unsigned)nqt), stream);
    else
      launch_fwd_p<true>(a, D, dim3(heads, (unsigned)nqt), stream);
  } else {
    FwdArgs b = a;
    b.xo = xcd_order(a.L.nseg, a.L.Hkv, a.L.group, nqt, a.causal != 0);
    launch_fwd_p<false>(b, D, dim3((unsigned)xcd_grid(b.xo)), stream);
  }
  return hipGetLastError();
}

}  // namespace attn
