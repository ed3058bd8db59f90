// Device-side building blocks shared by the attention kernels (gfx950 / CDNA4).
//
// Register layouts used throughout (64-lane wavefront, lane l):
//   v_mfma_f32_32x32x16_bf16  D[32x32] += A[32x16] * B[16x32]
//     A: lane l holds A[m = l%32][k = 8*(l/32) + j], j = 0..7
//     B: lane l holds B[k = 8*(l/32) + j][n = l%32]
//     C/D: lane l, register i holds C[m = 8*(i/4) + 4*(l/32) + i%4][n = l%32]
//   ds_read_b64_tr_b16 (transposing LDS read, groups of 16 lanes): element j
//     of lane i is element i%4 of the 8 bytes addressed by lane 4*j + i/4.
//
// An accumulator tile whose row index runs over a contraction dimension (keys
// for P, queries for dS) is fed back to the next MFMA as its B operand without
// any data movement: the 16 k-slots of contraction step t are bound to
//   row(t, s) = 16*t + 4*(s/8) + 8*((s%8)/4) + s%4,     s = 0..15,
// which is exactly the set of rows held in registers 8t..8t+7 of each lane.
// The matching A operand is read from a row-major LDS tile with two
// transposing reads (lds_tr8 below).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mw {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef short i16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
typedef uint16_t bf16_t;  // storage type of bf16 in global memory

#define MW_LDS __attribute__((address_space(3)))

__device__ __forceinline__ f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ f32x16 zero16() {
  f32x16 z;
#pragma unroll
  for (int i = 0; i < 16; ++i) z[i] = 0.f;
  return z;
}

// 2^x with the hardware instruction (v_exp_f32): results below the normal range
// flush to 0, which is harmless for softmax weights.  2^-inf = 0.
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// True if `pred` holds in any lane of the wavefront (a wave-uniform value).
__device__ __forceinline__ bool wave_any(bool pred) { return __builtin_amdgcn_ballot_w64(pred) != 0; }

// fp32 -> bf16, round to nearest even (finite inputs; +-inf map to +-inf).
__device__ __forceinline__ __bf16 to_bf16(float x) { return (__bf16)x; }

// 8 fp32 accumulator values (registers 8t..8t+7) -> one bf16x8 B operand.
__device__ __forceinline__ bf16x8 pack8(const f32x16& c, int t) {
  bf16x8 r;
#pragma unroll
  for (int j = 0; j < 8; ++j) r[j] = to_bf16(c[8 * t + j]);
  return r;
}

// ---------------------------------------------------------------------------
// LDS tiles: [rows][D] bf16, row-major, with the 16-byte slots of each row
// permuted by an XOR swizzle so that both access patterns used by the kernels
// spread over all banks:
//   - row reads: lane l reads 16 bytes of row l%32 (MFMA A/B operands);
//   - transposing reads: 8 consecutive rows x 64 bytes per instruction.
// ---------------------------------------------------------------------------
//
// D = 72 (nine slots, not a power of two) keeps rows dense and unswizzled:
// rows 144 bytes (36 banks) apart already put 16 consecutive rows on disjoint
// banks.  Its MFMA steps run over 80 (QK^T) and 96 (PV) columns; the columns
// past 72 read the next row (or the slack after the tile) and meet zeros in
// the register operand or land in output columns that are never stored.
template <int D>
struct Tile {
  static_assert(D == 64 || D == 72 || D == 128, "head dimension");
  static constexpr int SLOTS = D / 8;  // 16-byte slots per row
  __device__ __forceinline__ static int swz(int row) {
    if constexpr (D == 128) {
      return 4 * (row & 3) + ((row >> 2) & 3);
    } else if constexpr (D == 64) {
      const int u = row >> 1;
      return 4 * (u & 1) + ((u >> 1) & 3);
    } else {
      (void)row;
      return 0;
    }
  }
  // element offset of (row, col); col % 4 must be 0 for 8-byte and col % 8 for 16-byte access
  __device__ __forceinline__ static int off(int row, int col) {
    return row * D + ((((col >> 3) ^ swz(row)) << 3) | (col & 7));
  }
};

// 16-byte load of the A/B operand "row r, columns c..c+7" from an LDS tile.
template <int D>
__device__ __forceinline__ bf16x8 lds_row8(const bf16_t* tile, int r, int c) {
  return *reinterpret_cast<const bf16x8*>(tile + Tile<D>::off(r, c));
}

// A operand [m = column of the tile][k = slot] for contraction step t, taken
// from an LDS tile whose rows are the contraction index:
//   lane l gets tile[row(t, 8*(l/32) + j)][c0 + l%32], j = 0..7,
// with row() the slot binding described at the top of this file.  `rbase` is
// the tile row of slot row 0 (a multiple of 32 plus 16*t is added inside).
template <int D>
__device__ __forceinline__ bf16x8 lds_tr8(const bf16_t* tile, int rbase, int t, int c0, int lane) {
  const int rr = rbase + 16 * t + 4 * (lane >> 5) + ((lane & 15) >> 2);
  const int cc = c0 + 16 * ((lane >> 4) & 1) + 4 * (lane & 3);
  const bf16_t* p0 = tile + Tile<D>::off(rr, cc);
  const bf16_t* p1 = tile + Tile<D>::off(rr + 8, cc);
  i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((MW_LDS i16x4*)(p0));
  i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((MW_LDS i16x4*)(p1));
  bf16x8 r;
  bf16x4 lo4 = __builtin_bit_cast(bf16x4, lo);
  bf16x4 hi4 = __builtin_bit_cast(bf16x4, hi);
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    r[j] = lo4[j];
    r[4 + j] = hi4[j];
  }
  return r;
}

// Per-lane element offsets of a wave's fragment reads from an LDS tile, for
// kernels that compute them once: the row read of lds_row8 (row l % 32,
// columns 16 kk + 8 (l / 32)) per 16-column step kk, and the two transposing
// reads of lds_tr8 (rows rr and rr + 8, column block db).  The slot swizzle
// repeats every 16 rows, so a read of rows further down the tile (a later
// 32-row block, the second 16-row contraction step) is the same register plus
// a constant offset that the compiler folds into the instruction.
template <int D>
struct FragOffsets {
  static constexpr int KK = (D + 15) / 16, DB = (D + 31) / 32;
  int row[KK], tr[DB][2];
  __device__ __forceinline__ FragOffsets(int lane, int extra) {
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) row[kk] = Tile<D>::off(lane & 31, 16 * kk + 8 * (lane >> 5)) + extra;
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      const int rr = 4 * (lane >> 5) + ((lane & 15) >> 2);
      const int cc = db * 32 + 16 * ((lane >> 4) & 1) + 4 * (lane & 3);
      tr[db][0] = Tile<D>::off(rr, cc) + extra;
      tr[db][1] = Tile<D>::off(rr + 8, cc) + extra;
    }
  }
  // lds_row8(tile, rbase + l % 32, 16 kk + 8 (l / 32)), rbase a multiple of 16
  __device__ __forceinline__ bf16x8 row8(const bf16_t* tile, int rbase, int kk) const {
    return *reinterpret_cast<const bf16x8*>(tile + row[kk] + rbase * D);
  }
  // lds_tr8(tile, rbase, t, 32 db, l), rbase a multiple of 16
  __device__ __forceinline__ bf16x8 tr8(const bf16_t* tile, int rbase, int t, int db) const;
};

// The same A operand from the two addresses lds_tr8 computes (rows rr and
// rr + 8 of the tile at column cc), for callers that precompute them.
__device__ __forceinline__ bf16x8 lds_tr8_at(const bf16_t* p0, const bf16_t* p1) {
  i16x4 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((MW_LDS i16x4*)(p0));
  i16x4 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((MW_LDS i16x4*)(p1));
  bf16x8 r;
  bf16x4 lo4 = __builtin_bit_cast(bf16x4, lo);
  bf16x4 hi4 = __builtin_bit_cast(bf16x4, hi);
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    r[j] = lo4[j];
    r[4 + j] = hi4[j];
  }
  return r;
}

template <int D>
__device__ __forceinline__ bf16x8 FragOffsets<D>::tr8(const bf16_t* tile, int rbase, int t, int db) const {
  return lds_tr8_at(tile + tr[db][0] + (rbase + 16 * t) * D, tile + tr[db][1] + (rbase + 16 * t) * D);
}

// ---------------------------------------------------------------------------
// Direct global -> LDS staging (global_load_lds_dwordx4): each lane's 16 bytes
// land at wave_base + 16 * lane (wave_base in M0), so the tile swizzle is
// applied on the source side: LDS chunk ci (16 bytes, row ci / SLOTS, physical
// slot ci % SLOTS) is fetched from logical slot (physical ^ swz(row)) of the
// source row.  No registers are used and nothing is written back to LDS.
//
// The instruction is issued through inline assembly on purpose: the compiler
// treats the builtin form as an LDS write that may alias every later LDS read,
// and so inserted a full vmcnt(0) wait before the current tile's reads, which
// serialised the next tile's load latency with this tile's math.  Here the
// kernels synchronise explicitly instead: wait_vmem() (all counters zero)
// followed by a workgroup barrier before any wave reads a staged buffer, and
// no wave issues a load into a buffer before the barrier that ends the reads
// of that buffer.  Compiler-inserted vmcnt waits stay correct: loads it does
// not know of can only make such waits longer.
// `row_ptr(r)` returns the global address of tile row r; it must always be a
// valid address (callers clamp rows past the end of the data).
// ---------------------------------------------------------------------------
// LDS byte address of a pointer into LDS: the low 32 bits of its generic
// address (the aperture base is the high half), without the null check of an
// address-space cast.
__device__ __forceinline__ unsigned lds_addr(const void* p) { return (unsigned)(uintptr_t)p; }

// This wave's byte offset in a staging round (64 lanes x 16 bytes per wave),
// as a wave-uniform (scalar) value.
__device__ __forceinline__ unsigned wave_stage_off(int tid) {
  return __builtin_amdgcn_readfirstlane((unsigned)(tid & ~63) * 16u);
}

// `lds_dst` is the wave-uniform LDS byte address of the wave's 64 x 16 bytes.
__device__ __forceinline__ void dma_lds_16(const void* src, unsigned lds_dst) {
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(src), "s"(lds_dst) : "m0", "memory");
}
__device__ __forceinline__ void dma_lds_4(const void* src, unsigned lds_dst) {
  asm volatile("s_mov_b32 m0, %1\n\tglobal_load_lds_dword %0, off" ::"v"(src), "s"(lds_dst) : "m0", "memory");
}

// Pieces of a ROWS x D tile staged by NT threads: whole rounds of NT, the last
// one partial when ROWS * D / 8 is not a multiple of NT (D = 72).  Pieces past
// the tile fetch row 0 again and land in the slack that follows the tile, so
// an LDS tile buffer holds stage_elems() elements.
template <int D, int ROWS, int NT>
struct StagePlan {
  static constexpr int SLOTS = D / 8;
  static constexpr int PIECES = ROWS * SLOTS;
  static constexpr int ROUNDS = (PIECES + NT - 1) / NT;
  static constexpr int ELEMS = ROUNDS * NT * 8 > ROWS * D + 32 ? ROUNDS * NT * 8 : ROWS * D + 32;
  static_assert(PIECES % NT == 0 || D == 72, "only D = 72 stages a partial round");
  // at D = 72 the last row's reads run 24 elements past the tile into the
  // slack, which the partial round's extra pieces fill with (finite) data
  static_assert(D != 72 || PIECES % NT != 0, "D = 72 needs a partial last round to fill the slack");
};
template <int D, int ROWS, int NT>
constexpr int stage_elems() {
  return D == 72 ? StagePlan<D, ROWS, NT>::ELEMS : ROWS * D;
}

template <int D, int ROWS, int NT, typename RowPtr>
__device__ __forceinline__ void stage_rows_direct(bf16_t* lds_tile, RowPtr row_ptr, int tid) {
  using SP = StagePlan<D, ROWS, NT>;
  constexpr int SLOTS = SP::SLOTS;
#pragma unroll
  for (int it = 0; it < SP::ROUNDS; ++it) {
    const int ci0 = it * NT + tid;
    const int ci = (SP::PIECES % NT == 0 || ci0 < SP::PIECES) ? ci0 : 0;  // past the tile: row 0 again, into the slack
    const int row = ci / SLOTS, ps = ci % SLOTS;
    const int ls = ps ^ Tile<D>::swz(row);
    const bf16_t* src = row_ptr(row) + ls * 8;
    dma_lds_16(src, lds_addr(lds_tile) + it * NT * 16 + wave_stage_off(tid));
  }
}

// The same load with a wave-uniform 64-bit base held in SGPRs and a per-lane
// 32-bit byte offset (the saddr form): a tile whose rows are equally spaced is
// staged from one scalar base per tile and offsets computed once per kernel.
__device__ __forceinline__ void dma_lds_16_s(const void* sbase, unsigned voff, unsigned lds_dst) {
  asm volatile("s_mov_b32 m0, %2\n\tglobal_load_lds_dwordx4 %0, %1" ::"v"(voff), "s"(sbase), "s"(lds_dst)
               : "m0", "memory");
}

// Byte offsets, from the tile's first row, of the 16-byte pieces this thread
// stages of a ROWS x D tile whose rows are `row_stride` elements apart (same
// piece assignment and swizzle as stage_rows_direct).  Computed once; the
// offsets must fit 32 bits (ROWS * row_stride * 2 < 2^32, checked by the host).
template <int D, int ROWS, int NT>
struct RowOffsets {
  static constexpr int SLOTS = D / 8;
  static constexpr int ROUNDS = StagePlan<D, ROWS, NT>::ROUNDS;
  unsigned off[ROUNDS];
  __device__ __forceinline__ RowOffsets(long long row_stride, int tid) {
#pragma unroll
    for (int it = 0; it < ROUNDS; ++it) {
      const int ci0 = it * NT + tid;
      const int ci = (StagePlan<D, ROWS, NT>::PIECES % NT == 0 || ci0 < StagePlan<D, ROWS, NT>::PIECES) ? ci0 : 0;
      const int row = ci / SLOTS, ps = ci % SLOTS;
      const int ls = ps ^ Tile<D>::swz(row);
      off[it] = (unsigned)((long long)row * row_stride * 2 + ls * 16);
    }
  }
};

// Stage a tile whose row 0 is at `tile` (wave-uniform) with rows laid out as
// `ro` describes.
template <int D, int ROWS, int NT>
__device__ __forceinline__ void stage_rows_s(bf16_t* lds_tile, const bf16_t* tile, const RowOffsets<D, ROWS, NT>& ro,
                                             int tid) {
#pragma unroll
  for (int it = 0; it < RowOffsets<D, ROWS, NT>::ROUNDS; ++it) {
    dma_lds_16_s(tile, ro.off[it], lds_addr(lds_tile) + it * NT * 16 + wave_stage_off(tid));
  }
}

// Same staging for a K tile and a V tile whose rows come from the same
// positions: row_src(row) returns the pair of row pointers, so the address
// arithmetic of a row is done once for both tiles.
struct RowPair {
  const bf16_t* k;
  const bf16_t* v;
};
template <int D, int ROWS, int NT, typename RowSrc>
__device__ __forceinline__ void stage_kv_rows_direct(bf16_t* k_tile, bf16_t* v_tile, RowSrc row_src, int tid) {
  using SP = StagePlan<D, ROWS, NT>;
  constexpr int SLOTS = SP::SLOTS;
#pragma unroll
  for (int it = 0; it < SP::ROUNDS; ++it) {
    const int ci0 = it * NT + tid;
    const int ci = (SP::PIECES % NT == 0 || ci0 < SP::PIECES) ? ci0 : 0;  // past the tile: row 0 again, into the slack
    const int row = ci / SLOTS, ps = ci % SLOTS;
    const int ls = ps ^ Tile<D>::swz(row);
    const RowPair src = row_src(row);
    const unsigned dst = it * NT * 16 + wave_stage_off(tid);
    dma_lds_16(src.k + ls * 8, lds_addr(k_tile) + dst);
    dma_lds_16(src.v + ls * 8, lds_addr(v_tile) + dst);
  }
}

// 64 consecutive fp32 values (rows r0..r0+63, clamped to n-1) into LDS by one wave.
__device__ __forceinline__ void stage_f32x64_direct(float* lds, const float* g, int r0, int n, int lane) {
  const float* src = g + min(r0 + lane, n - 1);
  dma_lds_4(src, lds_addr(lds));
}

// Wait until this wave's outstanding memory operations (global loads, including
// direct-to-LDS loads, and LDS accesses) have completed: s_waitcnt with every
// counter at zero.
__device__ __forceinline__ void wait_vmem() { __builtin_amdgcn_s_waitcnt(0); }

// Wait until at most n * P of this wave's vector-memory operations are
// outstanding (0 <= n <= NMAX <= 3, wave-uniform); the other counters are not
// waited on.  gfx9 encoding: vmcnt in bits 3:0 and 15:14, expcnt 6:4,
// lgkmcnt 11:8 (7 and 15: no wait).
template <int N>
__device__ __forceinline__ void waitcnt_vm() {
  static_assert(N >= 0 && N <= 63, "vmcnt is six bits");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}
template <int P, int NMAX>
__device__ __forceinline__ void wait_vmem_upto(int n) {
  static_assert(NMAX <= 3, "up to three groups outstanding");
  if constexpr (NMAX >= 3) {
    if (n >= 3) {
      waitcnt_vm<3 * P>();
      return;
    }
  }
  if constexpr (NMAX >= 2) {
    if (n >= 2) {
      waitcnt_vm<2 * P>();
      return;
    }
  }
  if constexpr (NMAX >= 1) {
    if (n >= 1) {
      waitcnt_vm<P>();
      return;
    }
  }
  waitcnt_vm<0>();
}


// Combine a value with the one held by lane l ^ 32: gfx950's permlane32 swap
// exchanges the two 32-lane halves of a register in the VALU, without the LDS
// round trip of a generic shuffle.  The two results are {x[l], x[l ^ 32]} in
// some order, so a symmetric combination needs no select.
__device__ __forceinline__ float max_halves(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float sum_halves(float x) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// XCD-aware order: consecutive workgroup ids are dealt round-robin to the 8
// XCDs; remap so that each XCD receives one contiguous range of logical work
// items (whole heads, heaviest query tiles first), which keeps a head's K/V in
// one XCD's L2.
__device__ __forceinline__ int xcd_remap(int bid, int n) {
  if (n % 8) return bid;
  return (bid % 8) * (n / 8) + bid / 8;
}

// Work item (batch*head, query tile, key split) of forward workgroup `bid` in a
// grid of n = BH * nqt * NS.  Later query tiles see more keys, so they go
// first.  When BH is a multiple of 8, each XCD (workgroup ids are dealt to
// the 8 XCDs round-robin) takes BH / 8 whole heads, and within them the query
// tiles run heaviest first across those heads: interleaving the heads evens
// out the XCD's finish (a simulation of the D = 64 training shape's dispatch
// gives a 23% shorter makespan than taking the heads one after another, each
// heaviest first).  Otherwise the XCD-aware order of xcd_remap, heads one
// after another.
// The same order for any tiling: workgroup `bid` of n = BH * ntiles * NS gets
// (batch*head, tile rank, split), rank 0 being the heaviest tile of its head.
__device__ __forceinline__ void tile_item(int bid, int n, int BH, int ntiles, int NS, int& bh, int& rank,
                                          int& split) {
  if (BH % 8 == 0) {
    const int x = bid % 8, local = bid / 8, hpx = BH / 8;
    const int r = local / (hpx * NS), rem = local - r * (hpx * NS);
    bh = x * hpx + rem / NS;
    rank = r;
    split = rem % NS;
  } else {
    const int logical = xcd_remap(bid, n);
    split = logical % NS;
    bh = (logical / NS) / ntiles;
    rank = (logical / NS) % ntiles;
  }
}

__device__ __forceinline__ void fwd_item(int bid, int n, int BH, int nqt, int NS, int& bh, int& qt, int& split) {
  int rank;
  tile_item(bid, n, BH, nqt, NS, bh, rank, split);
  qt = nqt - 1 - rank;
}
// Cached attention: the heads one after another on each XCD (xcd_remap).
// Within a head, first its n_whole heaviest query tiles, unsplit (nst = 1),
// heaviest first; then the remaining tiles over NS key ranges (nst = NS),
// split-major: every such tile's first key range (heaviest first), then every
// tile's second range, and so on, so that the workgroups an XCD runs at once
// read the same key range and a window larger than the L2 is streamed once
// per range.  Split-major measured 1-4% faster than keeping a query tile's
// splits adjacent or interleaving the heads.
__device__ __forceinline__ void cached_item(int bid, int n, int nqt, int NS, int n_whole, int& bh, int& qt, int& split,
                                            int& nst) {
  const int logical = xcd_remap(bid, n);
  const int light = nqt - n_whole;
  const int per_head = n_whole + light * NS;
  bh = logical / per_head;
  const int r = logical - bh * per_head;
  if (r < n_whole) {
    split = 0;
    nst = 1;
    qt = nqt - 1 - r;
  } else {
    const int s = r - n_whole;
    split = s / light;
    nst = NS;
    qt = light - 1 - (s - split * light);
  }
}

// Row (within a 32-row accumulator block) of accumulator register i in lane l.
__device__ __forceinline__ int acc_row(int i, int lane) { return 8 * (i >> 2) + 4 * (lane >> 5) + (i & 3); }

// ---------------------------------------------------------------------------
// Visibility of key j to query row i.  Three rules share one form: key j is
// visible iff j < e1 or s2 <= j < e2.
//   BLOCK_CAUSAL  : chunk c = i / L; e1 = min(T, (c+1) L); second range empty.
//   QUEUED_CAUSAL : queued chunk q = i / qlen; e1 = wL + (q+1) qlen.
//   QUEUED_ISOL   : e1 = wL; [s2, e2) = [wL + q qlen, wL + (q+1) qlen).
// Keys are positions in the (virtual) key sequence.
// ---------------------------------------------------------------------------
enum VisMode { VIS_BLOCK_CAUSAL = 0, VIS_QUEUED_CAUSAL = 1, VIS_QUEUED_ISOLATED = 2 };

struct Vis {
  int mode;
  int L;      // chunk length (training) / committed chunk length (cached)
  int Tk;     // number of keys
  int qlen;   // queued chunk length (cached)
  int wL;     // window tokens (cached)
  __device__ __forceinline__ void range(int i, int& e1, int& s2, int& e2) const {
    if (mode == VIS_BLOCK_CAUSAL) {
      const int c = i / L;
      e1 = min(Tk, (c + 1) * L);
      s2 = e1;
      e2 = e1;
    } else {
      const int qc = i / qlen;
      if (mode == VIS_QUEUED_CAUSAL) {
        e1 = wL + (qc + 1) * qlen;
        s2 = e1;
        e2 = e1;
      } else {
        e1 = wL;
        s2 = wL + qc * qlen;
        e2 = s2 + qlen;
      }
    }
  }
};

// Workgroups of `threads` threads running `kernel` that one CU holds at once,
// from the runtime's occupancy calculator (the kernel's registers and LDS as
// built), or `fallback` where the runtime cannot answer (no device present:
// the figure then only sizes a workspace).
template <typename Kernel>
inline int resident_workgroups(Kernel kernel, int threads, int fallback) {
  int n = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, kernel, threads, 0) != hipSuccess || n < 1) {
    (void)hipGetLastError();
    return fallback;
  }
  return n;
}

}  // namespace mw
