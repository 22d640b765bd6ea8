// Device-side building blocks shared by the attention kernels (gfx950).
//
// MFMA v_mfma_f32_32x32x16_bf16 operand conventions used throughout:
//   A (32 x 16): lane l holds row (l % 32), reduction slots k = 8*(l/32) + e
//                for its 8 bf16 elements e = 0..7;
//   B (16 x 32): lane l holds column (l % 32), the same reduction slots;
//   C (32 x 32): lane l holds column (l % 32) and, in accumulator element r,
//                row 8*(r/4) + 4*(l/32) + (r%4).
// Only the row/column placement and the identical slot assignment of A and B
// matter: any consistent relabelling of the reduction index gives the same
// sum, which is how accumulator tiles are fed back as B operands without a
// shuffle through LDS.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace attn {

typedef __attribute__((ext_vector_type(8))) __bf16 bf16x8;
typedef __attribute__((ext_vector_type(2))) __bf16 bf16x2;
typedef __attribute__((ext_vector_type(16))) float f32x16;
typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(4))) uint32_t u32x4;
typedef __attribute__((ext_vector_type(2))) uint32_t u32x2;

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;

__device__ __forceinline__ f32x16 mfma32(u32x4 a, u32x4 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(
      __builtin_bit_cast(bf16x8, a), __builtin_bit_cast(bf16x8, b), c, 0, 0, 0);
}

// Two fp32 -> packed bf16 pair (round to nearest even; v_cvt_pk_bf16_f32).
__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi) {
  bf16x2 v;
  v[0] = (__bf16)lo;
  v[1] = (__bf16)hi;
  return __builtin_bit_cast(uint32_t, v);
}

__device__ __forceinline__ float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// Accumulator elements 8*c .. 8*c+7 of a 32x32 tile as a bf16 B operand.
__device__ __forceinline__ u32x4 pack_chunk(const f32x16& x, int c) {
  u32x4 r;
  r[0] = pack_bf16(x[8 * c + 0], x[8 * c + 1]);
  r[1] = pack_bf16(x[8 * c + 2], x[8 * c + 3]);
  r[2] = pack_bf16(x[8 * c + 4], x[8 * c + 5]);
  r[3] = pack_bf16(x[8 * c + 6], x[8 * c + 7]);
  return r;
}

__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Maximum and sum of x over the lane pair (l, l ^ 32), the same on both
// lanes.  v_permlane32_swap exchanges the two halves of the wavefront in the
// vector ALU (no LDS round trip, as a cross-lane shuffle would take); its
// two results hold the pair's two values, one each, so a symmetric
// combination of them is the pair's.
__device__ __forceinline__ float max_halves(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                  false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float sum_halves(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false,
                                                  false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

__device__ __forceinline__ u32x4 ld16(const uint16_t* p) { return *reinterpret_cast<const u32x4*>(p); }
__device__ __forceinline__ void st16(uint16_t* p, u32x4 v) { *reinterpret_cast<u32x4*>(p) = v; }
__device__ __forceinline__ void st8(uint16_t* p, u32x2 v) { *reinterpret_cast<u32x2*>(p) = v; }

// Wavefront index as a scalar (the compiler cannot prove threadIdx.x >> 6 is
// uniform, and a uniform value keeps wave-level decisions as scalar branches).
__device__ __forceinline__ int wave_id() { return __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6)); }

// ---------------------------------------------------------------------------
// Buffer loads: a resource over [base, base + bytes) makes out-of-range
// loads return zero in hardware, with no branch and no access.
// ---------------------------------------------------------------------------
typedef __amdgpu_buffer_rsrc_t rsrc_t;
constexpr int kRsrcFlags = 0x00020000;   // raw buffer, 32-bit data format (gfx9 family)

__device__ __forceinline__ rsrc_t make_rsrc(const void* base, int64_t bytes) {
  const int64_t lim = bytes < 0 ? 0 : (bytes > 0x7fffffff ? 0x7fffffff : bytes);
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)lim, kRsrcFlags);
}

__device__ __forceinline__ u32x4 bload16(rsrc_t r, int byte_off) {
  return __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(r, byte_off, 0, 0));
}

// Rows [row0, len) of one head as a buffer resource: loads of rows >= len
// (the tile tail) return zero.  row_stride in elements.
__device__ __forceinline__ rsrc_t rows_rsrc(const uint16_t* head_base, int row0, int len,
                                             int64_t row_stride) {
  return make_rsrc(head_base + (int64_t)row0 * row_stride,
                   (int64_t)(len - row0) * row_stride * 2);
}

// ---------------------------------------------------------------------------
// Asynchronous tiles: [64 rows][P] bf16 tiles (P = lds_pitch<D>() elements
// per row, D of them used) filled straight from global memory into LDS
// (buffer_load ... lds) and read back either row-major (16-byte MFMA operand
// rows) or transposed (ds_read_b64_tr_b16).  gfx950's LDS serves 64 banks x
// 4 bytes: a 16-byte access 16 lanes at a time, an 8-byte access 32 lanes at
// a time.
//
// A DMA load writes 16 bytes per lane to consecutive LDS addresses (lane L
// of the wave at base + 16 L), so the layout is chosen by which source chunk
// each lane fetches: LDS granule p holds row p / (P/8), logical 16-byte chunk
// (p % (P/8)) ^ tile_swz<P>(row).  The swizzle makes both read patterns hit
// 64 distinct banks per access phase: sixteen consecutive rows at one chunk
// (row-major reads), and four consecutive rows x four chunks (transposed
// reads).
// ---------------------------------------------------------------------------
#define ATTN_LDS __attribute__((address_space(3)))
typedef __attribute__((ext_vector_type(4))) short s16x4;

// LDS row pitch (elements) of a tile whose rows hold D values: rows of
// D = 96 are padded to 128 elements, so that they use the 16-chunk swizzle
// below; chunks 12..15 of such rows are never read.
template <int D>
constexpr int lds_pitch() {
  static_assert(D == 64 || D == 96 || D == 128, "head dimension");
  return D == 96 ? 128 : D;
}

// Swizzle of the 16-byte chunks of row r of a tile with pitch P elements.
template <int P>
__device__ __forceinline__ int tile_swz(int r) {
  static_assert(P == 64 || P == 128, "tile pitch");
  if constexpr (P == 128)
    return ((r & 3) << 2) | ((r >> 2) & 3);
  else
    return (((r >> 1) & 1) << 2) | ((r >> 2) & 3);
}

// Byte offset given to the DMA lanes of the pad chunks of a padded row: far
// beyond any buffer's range (at most 2^31 - 1 bytes), so the hardware range
// check turns the load into zeros without a memory access.
constexpr int kPadOffset = (int)0xFFFFFF00u;

template <int D, int NW = 4>
struct AsyncTile {
  static constexpr int P = lds_pitch<D>();   // LDS row pitch (elements)
  static constexpr int CPR = P / 8;          // 16-byte chunks per LDS row
  static constexpr int NJ = CPR / NW;        // DMA instructions per wavefront (64 rows)
  static constexpr int ELEMS = 64 * P;       // bf16 elements per tile
  static_assert(NJ * NW * 64 == 64 * CPR, "tile split");
  int goff[NJ];                              // this lane's source byte offset per instruction
  __device__ __forceinline__ AsyncTile(int wave, int lane, int row_bytes) {
#pragma unroll
    for (int j = 0; j < NJ; ++j) {
      const int p = (wave * NJ + j) * 64 + lane;
      const int row = p / CPR;
      const int logical = (p % CPR) ^ tile_swz<P>(row);
      goff[j] = logical < D / 8 ? row * row_bytes + 16 * logical : kPadOffset;
    }
  }
  // Enqueue this wavefront's share of a tile: rows [0, 64) of `src` into
  // `dst` (the tile base in LDS).
  __device__ __forceinline__ void load(rsrc_t src, uint16_t* dst, int wave) const {
    load_at(src, goff, dst, wave);
  }
  // The same with explicit per-lane source offsets (gathered rows).
  __device__ __forceinline__ void load_at(rsrc_t src, const int (&off)[NJ], uint16_t* dst,
                                          int wave) const {
#pragma unroll
    for (int j = 0; j < NJ; ++j)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(
          src, (ATTN_LDS void*)(dst + (wave * NJ + j) * 64 * 8), 16, off[j], 0, 0, 0);
  }
  // Tile row and logical 16-byte chunk that this lane copies in DMA
  // instruction j.
  static __device__ __forceinline__ int row_of(int wave, int j, int lane) {
    return ((wave * NJ + j) * 64 + lane) / CPR;
  }
  static __device__ __forceinline__ int chunk_of(int wave, int j, int lane) {
    const int p = (wave * NJ + j) * 64 + lane;
    return (p % CPR) ^ tile_swz<P>(p / CPR);
  }
  // Source offset of instruction j when the tile's rows are gathered: row r
  // of the tile is row page[r] of a cache whose rows are row_bytes apart.
  // Invalid rows (ok false, or page outside [0, num_pages)) and pad chunks
  // read zeros.
  static __device__ __forceinline__ int gather_off(int wave, int j, int lane, int page, bool ok,
                                                   int num_pages, int row_bytes) {
    const int c = chunk_of(wave, j, lane);
    ok = ok && (unsigned)page < (unsigned)num_pages && c < D / 8;
    return ok ? page * row_bytes + 16 * c : kPadOffset;
  }
};

__device__ __forceinline__ int bload4(rsrc_t r, int byte_off) {
  return __builtin_amdgcn_raw_buffer_load_b32(r, byte_off, 0, 0);
}

// Row-major read offsets (elements) of an MFMA operand over rows
// 32*b + (lane % 32), 16-byte chunk 2c + half: rm[c] + 32*b*P.
template <int D>
struct RowReader {
  static constexpr int P = lds_pitch<D>();
  int rm[D / 16];
  __device__ __forceinline__ RowReader(int l32, int half) {
    const int x = tile_swz<P>(l32);
#pragma unroll
    for (int c = 0; c < D / 16; ++c) rm[c] = l32 * P + 8 * ((2 * c + half) ^ x);
  }
};

// Transposed reads: the A operand of a 32x32x16 MFMA whose row index is a
// column of the tile (d) and whose reduction index runs over tile rows.  For
// column block db and 16-row chunk c, lane (l32, half) receives rows
// 16c + 8(e/4) + 4 half + e%4 (e = 0..7) of column 32 db + l32, as two
// ds_read_b64_tr_b16 at tr[db][0] + 16 c P and tr[db][1] + 16 c P.
// (Within each 16-lane group, transposed read lane i returns element i % 4
// of the 8 bytes addressed by lanes 4e + i/4, e = 0..3.)
template <int D>
struct TransReader {
  static constexpr int P = lds_pitch<D>();
  int tr[D / 32][2];
  __device__ __forceinline__ TransReader(int lane) {
    const int grp = lane >> 4, j = lane & 15;
    const int g = grp & 1, h = grp >> 1, e = j >> 2, m = j & 3;
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) {
        const int row = 8 * hh + 4 * h + e;
        const int phys = (4 * db + 2 * g + (m >> 1)) ^ tile_swz<P>(row);
        tr[db][hh] = row * P + 8 * phys + 4 * (m & 1);
      }
  }
};

__device__ __forceinline__ u32x2 ld_tr(const uint16_t* p) {
  return __builtin_bit_cast(u32x2, __builtin_amdgcn_ds_read_tr16_b64_v4i16((ATTN_LDS s16x4*)(p)));
}

// Wait until at most N vector-memory operations of this wavefront are in
// flight (expcnt and lgkmcnt unconstrained).
template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | (7 << 4) | (15 << 8) | ((N >> 4) << 14));
}

// ---------------------------------------------------------------------------
// DMA through inline assembly, for tiles in a ring of LDS stages selected at
// run time: the compiler does not model these loads as LDS writes, so it
// adds no conservative waits before LDS reads of other stages.  Callers
// order them explicitly (wait_vm + barrier before a stage is read, a barrier
// after its last read before it is refilled).
// ---------------------------------------------------------------------------
typedef __attribute__((ext_vector_type(4))) int i32x4;

// Raw buffer descriptor over [base, base + bytes) (gfx9 layout: 48-bit base,
// stride 0, num_records, raw 32-bit data format).
__device__ __forceinline__ i32x4 make_desc(const void* base, int64_t bytes) {
  const uint64_t a = reinterpret_cast<uint64_t>(base);
  const int64_t lim = bytes < 0 ? 0 : (bytes > 0x7fffffff ? 0x7fffffff : bytes);
  i32x4 d;
  d[0] = (int)(uint32_t)a;
  d[1] = (int)((uint32_t)(a >> 32) & 0xffffu);
  d[2] = (int)lim;
  d[3] = kRsrcFlags;
  return d;
}

__device__ __forceinline__ i32x4 rows_desc(const void* head_base, int row0, int len,
                                           int64_t row_stride_bytes) {
  return make_desc(static_cast<const char*>(head_base) + (int64_t)row0 * row_stride_bytes,
                   (int64_t)(len - row0) * row_stride_bytes);
}

// A raw buffer descriptor over `bytes` bytes at `base`; bytes in [0, 2^31).
__device__ __forceinline__ i32x4 raw_desc(const char* base, int bytes) {
  const uint64_t a = reinterpret_cast<uint64_t>(base);
  return i32x4{(int)(uint32_t)a, (int)((uint32_t)(a >> 32) & 0xffffu), bytes, kRsrcFlags};
}

// Rows [row0, len) of a tensor whose rows are rb bytes apart, from `base`
// (its row 0), with 0 <= row0 < len and rb < 2^24: 32-bit products only,
// the range capped at cap_rows = (2^31 - 1) / rb whole rows.
__device__ __forceinline__ i32x4 rows_desc_rb(const char* base, int row0, int len, int rb,
                                              int cap_rows) {
  return raw_desc(base + (int64_t)row0 * rb, min(len - row0, cap_rows) * rb);
}

// The same rows as a buffer resource for the compiler's buffer builtins.
__device__ __forceinline__ rsrc_t rows_rsrc_rb(const char* base, int row0, int len, int rb,
                                               int cap_rows) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<char*>(base) + (int64_t)row0 * rb, (short)0,
                                           min(len - row0, cap_rows) * rb, kRsrcFlags);
}

// LDS byte address of a __shared__ object.
__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)(ATTN_LDS const void*)p;
}

// 16-byte-per-lane DMAs written as inline assembly, so that the compiler's
// wait insertion does not count them (the kernels wait for them explicitly).
// The LDS destination of buffer_load ... lds comes from M0; on the gfx9
// family an LDS DMA needs one wait state after an SALU write of M0, hence
// the s_nop after each write.  M0 is saved and restored around each block.
//
// One DMA: lane L's 16 bytes at byte voff of the buffer go to LDS byte
// lds_base + 16 L.
__device__ __forceinline__ void dma16(i32x4 desc, uint32_t lds_base, int voff) {
  uint32_t saved;
  lds_base = __builtin_amdgcn_readfirstlane(lds_base);
  asm volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %1\n\t"
      "s_nop 0\n\t"
      "buffer_load_dwordx4 %2, %3, 0 offen lds\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "s"(lds_base), "v"(voff), "s"(desc)
      : "memory");
}

// NJ DMAs in one block (NJ = 1, 2 or 4): DMA j takes byte voff[j] of the
// buffer to LDS byte lds_base + 1024 j + 16 L; M0 is set once and stepped
// by 1 KiB.
template <int NJ>
__device__ __forceinline__ void dma16_n(i32x4 desc, uint32_t lds_base, const int (&voff)[NJ]) {
  if constexpr (NJ == 1) {
    dma16(desc, lds_base, voff[0]);
  } else if constexpr (NJ == 2) {
    uint32_t saved;
    lds_base = __builtin_amdgcn_readfirstlane(lds_base);
    asm volatile(
        "s_mov_b32 %0, m0\n\t"
        "s_mov_b32 m0, %1\n\t"
        "s_nop 0\n\t"
        "buffer_load_dwordx4 %2, %4, 0 offen lds\n\t"
        "s_add_u32 m0, m0, 0x400\n\t"
        "s_nop 0\n\t"
        "buffer_load_dwordx4 %3, %4, 0 offen lds\n\t"
        "s_mov_b32 m0, %0"
        : "=&s"(saved)
        : "s"(lds_base), "v"(voff[0]), "v"(voff[1]), "s"(desc)
        : "memory", "scc");
  } else {
    static_assert(NJ == 4, "1, 2 or 4 DMAs per block");
    uint32_t saved;
    lds_base = __builtin_amdgcn_readfirstlane(lds_base);
    asm volatile(
        "s_mov_b32 %0, m0\n\t"
        "s_mov_b32 m0, %1\n\t"
        "s_nop 0\n\t"
        "buffer_load_dwordx4 %2, %6, 0 offen lds\n\t"
        "s_add_u32 m0, m0, 0x400\n\t"
        "s_nop 0\n\t"
        "buffer_load_dwordx4 %3, %6, 0 offen lds\n\t"
        "s_add_u32 m0, m0, 0x400\n\t"
        "s_nop 0\n\t"
        "buffer_load_dwordx4 %4, %6, 0 offen lds\n\t"
        "s_add_u32 m0, m0, 0x400\n\t"
        "s_nop 0\n\t"
        "buffer_load_dwordx4 %5, %6, 0 offen lds\n\t"
        "s_mov_b32 m0, %0"
        : "=&s"(saved)
        : "s"(lds_base), "v"(voff[0]), "v"(voff[1]), "v"(voff[2]), "v"(voff[3]), "s"(desc)
        : "memory", "scc");
  }
}

// This wavefront's share of a tile (instructions wave NJ .. wave NJ + NJ - 1
// of the tile's copy, 1 KiB of LDS each).
template <int D, int NW>
__device__ __forceinline__ void dma_tile(const AsyncTile<D, NW>& t, i32x4 desc, uint32_t tile_base,
                                         int wave) {
  constexpr int NJ = AsyncTile<D, NW>::NJ;
  dma16_n<NJ>(desc, tile_base + (uint32_t)(wave * NJ * 64 * 16), t.goff);
}

// Wait for this wavefront's vector-memory operations, including the DMAs
// above, which the compiler does not count.
__device__ __forceinline__ void wait_vm_all() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

// Wait until at most N of them are in flight (loads complete in order).
template <int N>
__device__ __forceinline__ void wait_vm_upto() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  asm volatile("s_waitcnt vmcnt(%0)" ::"n"(N) : "memory");
}

// Resolve segment z of a layout: first row offset (elements) and length.
// Packed offsets are clamped into [0, total] so a malformed cu_seqlens array
// cannot move any access outside the tensors.
struct Segment {
  int start;   // first row (packed) or 0
  int len;     // rows in this segment
};

// Keys of segment z of a paged layout: offsets into the page-index array,
// clamped into [0, nnz].
template <typename LayoutT>
__device__ __forceinline__ Segment kv_segment_of(const LayoutT& L, int z) {
  int a = L.kv_cu[z], b = L.kv_cu[z + 1];
  a = a < 0 ? 0 : (a > L.nnz ? L.nnz : a);
  b = b < a ? a : (b > L.nnz ? L.nnz : b);
  return Segment{a, b - a};
}

template <typename LayoutT>
__device__ __forceinline__ Segment segment_of(const LayoutT& L, int z) {
  Segment s;
  if (L.cu) {
    int a = L.cu[z], b = L.cu[z + 1];
    a = a < 0 ? 0 : (a > L.total ? L.total : a);
    b = b < a ? a : (b > L.total ? L.total : b);
    s.start = a;
    s.len = b - a;
    if (s.len > L.S) s.len = L.S;
  } else {
    s.start = 0;
    s.len = L.S;
  }
  return s;
}

}  // namespace attn
