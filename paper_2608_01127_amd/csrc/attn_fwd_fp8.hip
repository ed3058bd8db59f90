// fp8 (OCP e4m3) cached chunk attention at head width 128, and the fp8
// quantizer (gfx950).
//
// The low-precision inference variant follows the deployment direction the
// paper names in its conclusion (quantization to cut inference cost, Sec. 6);
// the attention it computes is the cached chunk attention of Sec. 3.5 (queued
// in-flight chunks over [sink | window | queued keys]).  Q, K and V are e4m3
// with per-tensor scales (value = code * scale); scores and probabilities are
// accumulated in fp32, and the probabilities are rounded to e4m3 (RNE) before
// the PV product.  Both products run on v_mfma_f32_32x32x64_f8f6f4, which has
// twice the bf16 rate and halves K/V bytes.
//
// Layouts (64-lane wave, lane l, h = l / 32):
//   S^T = K Q^T, contraction over d in two steps of 64: lane l supplies bytes
//     d = 64 kk + 32 h + 0..31 of key row l % 32 (A) and of query row l % 32
//     (B).  The instruction pairs byte j of A with byte j of B for every lane
//     half, so any common assignment of d to bytes is a valid contraction.
//   O^T += V^T P^T over the tile's 64 keys: byte j of lane l's B operand is
//     P of key kappa(h, j) = 32 (j / 16) + 8 ((j % 16) / 4) + 4 h + j % 4, which
//     is the accumulator layout of the two 32-key S^T blocks, so the
//     probabilities are packed without data movement; the A operand holds
//     V[kappa(h, j)][d] for d = 32 db + l % 32, read from the row-major V tile
//     with four transposing reads ds_read_b64_tr_b8 (in each group of 16 lanes,
//     byte j of lane i is byte i % 8 of the 8 bytes addressed by lane
//     2 j + (i % 16) / 8).
#include <algorithm>
#include <cmath>
#include <type_traits>

#include "mw_device.h"
#include "mw_kernels.h"

namespace mw {

typedef int i32x8 __attribute__((ext_vector_type(8)));
typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef int i32x2 __attribute__((ext_vector_type(2)));
typedef uint8_t fp8_t;

namespace {

constexpr int DH = 128;  // head width = bytes per fp8 row
constexpr float kE4m3Max = 448.f;

__device__ __forceinline__ f32x16 mfma_fp8(i32x8 a, i32x8 b, f32x16 c) {
  // formats 0/0: e4m3 x e4m3; block scales unused (the plain instruction)
  return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a, b, c, 0, 0, 0, 0, 0, 0);
}

// [rows][128] bytes with the 16-byte slots of row r permuted by
// swz(r) = (r & 7) ^ 4 ((r >> 3) & 1): eight consecutive rows hit eight
// different slots (the K row reads), and so do the rows {4h + 0..3, 8 + 4h +
// 0..3} of one transposing read (the V reads).
struct Tile8 {
  __device__ __forceinline__ static int swz(int row) { return (row & 7) ^ (((row >> 3) & 1) << 2); }
  __device__ __forceinline__ static int off(int row, int col) {
    return row * DH + ((((col >> 4) ^ swz(row)) << 4) | (col & 15));
  }
};

// K fragment of contraction step kk: K[row][64 kk + 32 h + 0..31].
__device__ __forceinline__ i32x8 lds_k8(const fp8_t* tile, int row, int kk, int lane) {
  const int c = 64 * kk + 32 * (lane >> 5);
  const i32x4 a = *reinterpret_cast<const i32x4*>(tile + Tile8::off(row, c));
  const i32x4 b = *reinterpret_cast<const i32x4*>(tile + Tile8::off(row, c + 16));
  return i32x8{a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
}

// V^T fragment of column block db over the 64 keys of `tile` (row 0 = first key).
__device__ __forceinline__ i32x8 lds_v8(const fp8_t* tile, int db, int lane) {
  const int lam = lane & 15;
  const int col = 32 * db + 16 * ((lane >> 4) & 1) + 8 * (lam & 1);
  const int rsub = 8 * (lam >> 3) + 4 * (lane >> 5) + ((lam >> 1) & 3);
  i32x8 r;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    const i32x2 x = __builtin_amdgcn_ds_read_tr8_b64_v2i32((MW_LDS i32x2*)(tile + Tile8::off(16 * q + rsub, col)));
    r[2 * q] = x[0];
    r[2 * q + 1] = x[1];
  }
  return r;
}

// Probabilities of two 32-key accumulator blocks -> e4m3 B operand (RNE; the
// values lie in [0, 2^8], inside the e4m3 range).  Each conversion writes one
// 16-bit half of its destination and keeps the other; the high-half
// conversion overwrites what the low-half one kept, so the low-half one takes
// its first input's register as the kept value instead of a zeroed register
// (a zero costs a move each).
__device__ __forceinline__ i32x8 pack_p8(const f32x16& s0, const f32x16& s1) {
  i32x8 r;
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    int x = __builtin_amdgcn_cvt_pk_fp8_f32(s0[4 * w], s0[4 * w + 1], __float_as_int(s0[4 * w]), false);
    r[w] = __builtin_amdgcn_cvt_pk_fp8_f32(s0[4 * w + 2], s0[4 * w + 3], x, true);
    x = __builtin_amdgcn_cvt_pk_fp8_f32(s1[4 * w], s1[4 * w + 1], __float_as_int(s1[4 * w]), false);
    r[4 + w] = __builtin_amdgcn_cvt_pk_fp8_f32(s1[4 * w + 2], s1[4 * w + 3], x, true);
  }
  return r;
}

// Byte offsets of the 16-byte pieces this thread stages of a ROWS x 128-byte
// tile whose rows are `row_stride` bytes apart (LDS piece ci = row ci / 8,
// physical slot ci % 8, fetched from logical slot (ci % 8) ^ swz(row)).
template <int ROWS, int NT>
struct RowOffsets8 {
  static constexpr int PIECES = ROWS * 8;
  static_assert(PIECES % NT == 0, "whole staging rounds");
  static constexpr int ROUNDS = PIECES / NT;
  unsigned off[ROUNDS];
  __device__ __forceinline__ RowOffsets8(long long row_stride, int tid) {
#pragma unroll
    for (int it = 0; it < ROUNDS; ++it) {
      const int ci = it * NT + tid;
      const int row = ci >> 3;
      off[it] = (unsigned)((long long)row * row_stride + 16 * ((ci & 7) ^ Tile8::swz(row)));
    }
  }
};

template <int ROWS, int NT>
__device__ __forceinline__ void stage8_s(fp8_t* lds_tile, const fp8_t* tile, const RowOffsets8<ROWS, NT>& ro, int tid) {
#pragma unroll
  for (int it = 0; it < RowOffsets8<ROWS, NT>::ROUNDS; ++it)
    dma_lds_16_s(tile, ro.off[it], lds_addr(lds_tile) + it * NT * 16 + wave_stage_off(tid));
}

struct RowPair8 {
  const fp8_t* k;
  const fp8_t* v;
};
template <int ROWS, int NT, typename RowSrc>
__device__ __forceinline__ void stage8_rows(fp8_t* k_tile, fp8_t* v_tile, RowSrc row_src, int tid) {
#pragma unroll
  for (int it = 0; it < ROWS * 8 / NT; ++it) {
    const int ci = it * NT + tid;
    const int row = ci >> 3;
    const int ls = (ci & 7) ^ Tile8::swz(row);
    const RowPair8 src = row_src(row);
    const unsigned dst = it * NT * 16 + wave_stage_off(tid);  // wave-uniform
    dma_lds_16(src.k + 16 * ls, lds_addr(k_tile) + dst);
    dma_lds_16(src.v + 16 * ls, lds_addr(v_tile) + dst);
  }
}

// One BN-key tile of the virtual key sequence [sink | window slots | queued]
// into LDS (same classification as the bf16 kernel: a tile inside the queued
// keys or inside one window chunk is staged from one base; tiles that straddle
// a boundary or the end map row by row; rows past the end read the last key).
// fp8 tensors are contiguous: queued [BH, Tq, 128], sink [BH, sink_len, 128],
// slots [S][BH, L, 128].
template <int BN, int NT>
__device__ __forceinline__ void stage_kv8(const FwdParams& p, int bh, int k0, fp8_t* Kt, fp8_t* Vt,
                                          const RowOffsets8<BN, NT>& ro, int tid) {
  const fp8_t* qk = reinterpret_cast<const fp8_t*>(p.k) + (long long)bh * p.Tq * DH;
  const fp8_t* qv = reinterpret_cast<const fp8_t*>(p.v) + (long long)bh * p.Tq * DH;
  const fp8_t* ks = reinterpret_cast<const fp8_t*>(p.k_slots);
  const fp8_t* vs = reinterpret_cast<const fp8_t*>(p.v_slots);
  const int kl = min(k0 + BN, p.Tk) - 1;
  const int kw0 = k0 - p.sink_len;
  const int w0 = kw0 > 0 ? kw0 / p.L : 0;
  const int off0 = kw0 - w0 * p.L;
  if (k0 >= p.wL && k0 + BN <= p.Tk) {  // queued keys only
    const long long j = k0 - p.wL;
    stage8_s<BN, NT>(Kt, qk + j * DH, ro, tid);
    stage8_s<BN, NT>(Vt, qv + j * DH, ro, tid);
    return;
  }
  // window keys rotated on load come from p.k_win (window order), values
  // always from the slots
  const fp8_t* kw = p.k_win;
  if (kw0 >= 0 && kl < p.wL && off0 + (kl - k0) < p.L) {  // one window chunk
    int slot = p.first_slot + w0;
    slot = slot >= p.S ? slot - p.S : slot;
    const long long in_chunk = ((long long)bh * p.L + off0) * DH;
    const long long e = (long long)slot * p.slot_stride + in_chunk;
    stage8_s<BN, NT>(Kt, kw != nullptr ? kw + (long long)w0 * p.slot_stride + in_chunk : ks + e, ro, tid);
    stage8_s<BN, NT>(Vt, vs + e, ro, tid);
    return;
  }
  stage8_rows<BN, NT>(Kt, Vt, [&](int r) -> RowPair8 {
    const int key = min(k0 + r, p.Tk - 1);
    if (key < p.sink_len) {
      const long long e = ((long long)bh * p.sink_len + key) * DH;
      return {reinterpret_cast<const fp8_t*>(p.k_sink) + e, reinterpret_cast<const fp8_t*>(p.v_sink) + e};
    }
    if (key < p.wL) {
      int w = w0, off = key - p.sink_len - w0 * p.L;
      while (off >= p.L) {  // at most one step when L >= BN
        off -= p.L;
        ++w;
      }
      int slot = p.first_slot + w;
      slot = slot >= p.S ? slot - p.S : slot;
      const long long in_chunk = ((long long)bh * p.L + off) * DH;
      const long long e = (long long)slot * p.slot_stride + in_chunk;
      return {kw != nullptr ? kw + (long long)w * p.slot_stride + in_chunk : ks + e, vs + e};
    }
    const long long j = key - p.wL;
    return {qk + j * DH, qv + j * DH};
  }, tid);
}

// RoPE re-shift of e4m3 keys when they are used (paper Sec. 3.5, re-indexing
// the retained window after an eviction), shared by the separate rotation pass
// and the rotation in the attention kernel's staging so that both produce the
// same bytes.  (cos, sin) of a rotation by -n positions of a pair whose
// one-position rotation is (c1, s1): (c1 - i s1)^n by repeated squaring in
// double (no device trigonometry; a relative error of a few 1e-15 for any n).
__device__ __forceinline__ void rope_cos_sin(long long n, double c1, double s1, float& c, float& s) {
  double br = c1, bi = n >= 0 ? -s1 : s1;
  n = n >= 0 ? n : -n;
  double cr = 1.0, ci = 0.0;
  while (n != 0) {  // at most 63 rounds
    if (n & 1) {
      const double t = cr * br - ci * bi;
      ci = cr * bi + ci * br;
      cr = t;
    }
    const double t = br * br - bi * bi;
    bi = 2.0 * br * bi;
    br = t;
    n >>= 1;
  }
  c = (float)cr;
  s = (float)ci;
}

// One 16-byte piece of a key row (pairs 8 pc .. 8 pc + 7; the band's pairs are
// p0 .. p0 + n_pairs - 1): each band pair is decoded, rotated in fp32 with the
// cos/sin of its band index, clamped to +-448 and rounded back to e4m3
// (nearest even, the quantizer's rounding).  The scale cancels: a rotation is
// linear, so codes are rotated as values.
__device__ __forceinline__ u32x4 rope_rotate_piece(u32x4 v, int pc, int p0, int n_pairs, const float* cosv,
                                                   const float* sinv) {
#pragma unroll
  for (int q = 0; q < 8; ++q) {
    const int pr = 8 * pc + q - p0;  // band pair index of this byte pair
    if (pr < 0 || pr >= n_pairs) continue;
    unsigned u = v[q / 2];
    // (the half selectors of the conversions are immediates; the clamp is one
    // median-of-three, equal to min(max(y, -448), 448) for the finite values
    // a rotation of e4m3 codes gives)
    const auto x = (q % 2) ? __builtin_amdgcn_cvt_pk_f32_fp8((int)u, true) : __builtin_amdgcn_cvt_pk_f32_fp8((int)u, false);
    const float c = cosv[pr], sn = sinv[pr];
    const float y0 = __builtin_amdgcn_fmed3f(fmaf(x[0], c, -x[1] * sn), -kE4m3Max, kE4m3Max);
    const float y1 = __builtin_amdgcn_fmed3f(fmaf(x[0], sn, x[1] * c), -kE4m3Max, kE4m3Max);
    u = (q % 2) ? (unsigned)__builtin_amdgcn_cvt_pk_fp8_f32(y0, y1, (int)u, true)
                : (unsigned)__builtin_amdgcn_cvt_pk_fp8_f32(y0, y1, (int)u, false);
    v[q / 2] = u;
  }
  return v;
}

constexpr float kRescaleThreshold8 = 8.f;  // probabilities stay <= 2^8 < 448

// NW waves of RB 32-row query blocks in KG key groups of NW / KG row waves;
// each step stages KG * BN keys (BN a multiple of 64) and group g works on
// its BN-key slice; the groups merge (m, l, O) through LDS at the end.  With
// key groups (the few-row configurations) the tiles stream four stages deep.
// ROT: the instantiation that rotates window keys with re-shifts pending in
// staging (rs), for calls with one query tile per head.
template <int NW, int RB, int BN, int KG, bool ROT>
__global__ __launch_bounds__(64 * NW, KG > 1 ? 1 : ((8 / NW) > 0 ? (8 / NW) : 1)) void attn_fwd_fp8_kernel(
    FwdParams p, const RopeStage rs) {  // (key-group configurations hold 132 KB of LDS: one workgroup per CU)
  static_assert(NW % KG == 0, "waves split evenly into key groups");
  constexpr int NWR = NW / KG;
  constexpr int BM = 32 * RB * NWR, NT = 64 * NW, KB = BN / 32, KP = BN / 64, BK = BN * KG;
  constexpr int KK = DH / 64, DB = DH / 32;
  constexpr int NSTG = KG > 1 ? 4 : 2;
  __shared__ __attribute__((aligned(16))) fp8_t lds[2][NSTG][BK * DH];  // K, V x stages
  fp8_t(*Ks)[BK * DH] = lds[0];
  fp8_t(*Vs)[BK * DH] = lds[1];

  const int NS = p.n_splits;  // key ranges of a split tile (partials layout)
  int bh, qt, split, nst;      // nst: key ranges of this workgroup's tile
  cached_item(blockIdx.x, gridDim.x, p.n_qtiles, NS, p.n_whole, bh, qt, split, nst);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int rw = wave % NWR, kg = wave / NWR;  // row wave, key group
  const int q0 = qt * BM;
  const int b_ = bh / p.H, h_ = bh - b_ * p.H;
  const fp8_t* qg = reinterpret_cast<const fp8_t*>(p.q) + (long long)bh * p.Tq * DH;

  Vis vis{p.vis_mode, p.L, p.Tk, p.qlen, p.wL};

  int qrow[RB], e1[RB], s2[RB], e2[RB];
  i32x8 qf[RB][KK];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    qrow[rb] = q0 + (rw * RB + rb) * 32 + (lane & 31);
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
      if constexpr (NSTG > 2) break;  // staged through LDS with the first K/V tiles
      if (qrow[rb] < p.Tq) {
        const fp8_t* src = qg + (long long)qrow[rb] * DH + 64 * kk + 32 * (lane >> 5);
        const i32x4 a = *reinterpret_cast<const i32x4*>(src);
        const i32x4 b = *reinterpret_cast<const i32x4*>(src + 16);
        qf[rb][kk] = i32x8{a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
      } else {
        qf[rb][kk] = i32x8{0, 0, 0, 0, 0, 0, 0, 0};
      }
    }
    vis.range(min(qrow[rb], p.Tq - 1), e1[rb], s2[rb], e2[rb]);
  }
  int e1f, s2f, e2f, e1l, s2l, e2l;
  vis.range(q0, e1f, s2f, e2f);
  vis.range(min(q0 + BM, p.Tq) - 1, e1l, s2l, e2l);
  const int kend_all = max(e1l, e2l);
  const int ntiles = (kend_all + BK - 1) / BK;
  const int kbeg = (int)((long long)ntiles * split / nst) * BK;
  const int kend = min(kend_all, (int)((long long)ntiles * (split + 1) / nst) * BK);
  auto advance = [&](int k) {
    int n = k + BK;
    if (n >= e1l && n + BK <= s2f) n = (s2f / BK) * BK;
    return n;
  };

  f32x16 o[RB][DB];
  float m[RB], lsum[RB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
#pragma unroll
    for (int db = 0; db < DB; ++db) o[rb][db] = zero16();
    m[rb] = -INFINITY;
    lsum[rb] = 0.f;
  }
  const float c = p.scale_log2;  // softmax scale * q_scale * k_scale * log2(e)
  const int kfull = max(0, (e1f / BK) * BK);

  auto step = [&](auto masked, const int k0, const fp8_t* Kt, const fp8_t* Vt) {
    f32x16 s[RB][KB];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) s[rb][kb] = zero16();
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) {
        const i32x8 kfrag = lds_k8(Kt, kb * 32 + (lane & 31), kk, lane);
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) s[rb][kb] = mfma_fp8(kfrag, qf[rb][kk], s[rb][kb]);
      }
    }
    if constexpr (decltype(masked)::value) {
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) {
#pragma unroll
        for (int kb = 0; kb < KB; ++kb) {
#pragma unroll
          for (int i = 0; i < 16; ++i) {
            const int key = k0 + kb * 32 + acc_row(i, lane);
            const bool ok = (key < e1[rb]) | ((key >= s2[rb]) & (key < e2[rb]));  // no short circuit
            s[rb][kb][i] = ok ? s[rb][kb][i] : -INFINITY;
          }
        }
      }
    }
    float mx[RB];
    bool need_any = false;
    bool need[RB];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      mx[rb] = -INFINITY;
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) {
#pragma unroll
        for (int i = 0; i < 16; ++i) mx[rb] = fmaxf(mx[rb], s[rb][kb][i]);
      }
      mx[rb] = max_halves(mx[rb]) * c;
      need[rb] = mx[rb] > m[rb] + kRescaleThreshold8;
      need_any |= need[rb];
    }
    if (wave_any(need_any)) {
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) {
        const float alpha = need[rb] ? fast_exp2(m[rb] - mx[rb]) : 1.f;
        lsum[rb] *= alpha;
#pragma unroll
        for (int db = 0; db < DB; ++db) {
#pragma unroll
          for (int i = 0; i < 16; ++i) o[rb][db][i] *= alpha;
        }
        m[rb] = need[rb] ? mx[rb] : m[rb];
      }
    }
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      const float nm = (m[rb] == -INFINITY) ? 0.f : -m[rb];
      float ls = 0.f;
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) {
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          const float pv = fast_exp2(fmaf(s[rb][kb][i], c, nm));
          s[rb][kb][i] = pv;
          ls = (kb == 0 && i == 0) ? pv : ls + pv;  // (no add of the zero start)
        }
      }
      lsum[rb] += ls;
    }
#pragma unroll
    for (int kp = 0; kp < KP; ++kp) {
      i32x8 pb[RB];
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) pb[rb] = pack_p8(s[rb][2 * kp], s[rb][2 * kp + 1]);
#pragma unroll
      for (int db = 0; db < DB; ++db) {
        const i32x8 vfrag = lds_v8(Vt + kp * 64 * DH, db, lane);
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) o[rb][db] = mfma_fp8(vfrag, pb[rb], o[rb][db]);
      }
    }
  };

  // Rotation in staging (window keys with re-shifts pending, calls the host
  // routes here): the window chunks this workgroup's key range spans (at most
  // kRopeStageChunks, chunks of at least BK / 2 keys, as the host checks) get a
  // cos/sin table of their band pairs in LDS, computed once the first tiles
  // are in flight; each staged K tile's window rows are rotated in place after
  // the tile lands, and a barrier publishes them.
  static_assert(NT % BK == 0 && (BK & (BK - 1)) == 0, "rotation maps a thread to one row of the tile");
  __shared__ float rtab[ROT ? kRopeStageChunks : 1][2][64];
  const bool rot = ROT && rs.n_pairs > 0;  // (ROT = false: an instantiation without the rotation code)
  int w_lo = 0, nwc = 0;
  if (rot) {
    const int a0 = max(kbeg, p.sink_len), a1 = min(((kend + BK - 1) / BK) * BK, p.wL);
    if (a0 < a1) {
      w_lo = (a0 - p.sink_len) / p.L;
      nwc = min((a1 - 1 - p.sink_len) / p.L - w_lo + 1, kRopeStageChunks);
    }
  }
  // window rows of the staged tile [k0, k0 + BK): their band pieces, rotated
  // in place, thread t on row t mod BK (a uniform test says whether the tile
  // has any); a tile spans at most three window chunks, whose first rows are
  // found once per tile
  auto rotate = [&](const int k0, const int buf) {
    if constexpr (!ROT) return false;
    const int r0 = max(p.sink_len - k0, 0), r1 = min(p.wL - k0, BK);
    if (r0 >= r1 || nwc == 0) return false;
    const int kw = k0 + r0 - p.sink_len;  // window index of row r0
    const int wa = kw / p.L;
    const int b1 = r0 + (wa + 1) * p.L - kw, b2 = b1 + p.L;  // first rows of the next two chunks
    const int pc0 = rs.dim_offset >> 4, pc1 = (rs.dim_offset + 2 * rs.n_pairs - 1) >> 4;
    const int row = tid & (BK - 1);
    if (row >= r0 && row < r1) {
      const int wi = min(max(wa - w_lo + (row >= b1) + (row >= b2), 0), nwc - 1);
      const int p0 = rs.dim_offset >> 1;
      fp8_t* kt = Ks[buf];
      // the thread's first two pieces with both reads in flight, then any more
      constexpr int G = NT / BK;
      const int pa = pc0 + tid / BK, pb = pa + G;
      u32x4* aa = reinterpret_cast<u32x4*>(kt + Tile8::off(row, 16 * min(pa, 7)));
      u32x4* ab = reinterpret_cast<u32x4*>(kt + Tile8::off(row, 16 * min(pb, 7)));
      const u32x4 va = *aa, vb = *ab;
      if (pa <= pc1) *aa = rope_rotate_piece(va, pa, p0, rs.n_pairs, rtab[wi][0], rtab[wi][1]);
      if (pb <= pc1) *ab = rope_rotate_piece(vb, pb, p0, rs.n_pairs, rtab[wi][0], rtab[wi][1]);
      for (int pc = pb + G; pc <= pc1; pc += G) {
        u32x4* a = reinterpret_cast<u32x4*>(kt + Tile8::off(row, 16 * pc));
        *a = rope_rotate_piece(*a, pc, p0, rs.n_pairs, rtab[wi][0], rtab[wi][1]);
      }
    }
    return true;
  };
  // the cos/sin table: lane i takes pair i's one-position rotation, read with
  // scalar loads (a vector load here would be the only one the compiler
  // tracks, and it would wait for the tiles in flight as well); wave w the
  // chunks w, w + NW, ...
  auto rope_table = [&]() {
    if constexpr (!ROT) return;
    if (!rot) return;
    double c1 = 1.0, s1 = 0.0;
    for (int i = 0; i < rs.n_pairs; ++i) {
      const double ci = rs.a.c1[i], si = rs.a.s1[i];
      c1 = lane == i ? ci : c1;
      s1 = lane == i ? si : s1;
    }
    for (int wi = __builtin_amdgcn_readfirstlane(wave); wi < nwc; wi += NW) {
      const long long n = rs.a.pend[w_lo + wi];
      if (lane < rs.n_pairs) rope_cos_sin(n, c1, s1, rtab[wi][0][lane], rtab[wi][1][lane]);
    }
  };
  // this wave's slice of a staged step: keys [kg * BN, (kg + 1) * BN)
  auto slice = [&](auto masked, const int k0, const int st) {
    step(masked, k0 + kg * BN, Ks[st] + kg * BN * DH, Vs[st] + kg * BN * DH);
  };
  const RowOffsets8<BK, NT> ro(DH, tid);
  int kc = advance(kbeg - BK);
  if constexpr (NSTG > 2) {
    // Up to NSTG - 1 tiles in flight: each wave waits on the vector-memory
    // counter only for the oldest of its tiles (a tile is 2 * ROUNDS loads per
    // thread on every staging path), then one barrier publishes the tile and
    // frees the buffer computed last for the next one.  The Q tile is staged
    // first, into the last stage buffer, which the first tiles leave free, and
    // read into registers before the loop's first barrier frees it (loaded
    // straight into registers, the compiler, blind to the LDS-direct loads,
    // would wait for all outstanding loads inside the loop).
    constexpr int P = 2 * RowOffsets8<BK, NT>::ROUNDS;
    constexpr int QR = BM * 8 / NT;  // Q staging rounds
    static_assert(P * (NSTG - 1) <= 63, "vector-memory counter range");
    static_assert((BM * 8) % NT == 0 && BM <= BK, "the Q tile is whole rounds and fits a K buffer");
    fp8_t* qs = Ks[NSTG - 1];
#pragma unroll
    for (int it = 0; it < QR; ++it) {
      const int ci = it * NT + tid;
      const int row = ci >> 3;
      const int ls = (ci & 7) ^ Tile8::swz(row);
      const fp8_t* src = qg + (long long)min(q0 + row, p.Tq - 1) * DH + 16 * ls;
      dma_lds_16(src, lds_addr(qs) + it * NT * 16 + wave_stage_off(tid));
    }
    int ki = kc, ib = 0, ahead = 0;  // next tile to issue, its buffer, tiles issued and not yet used
#pragma unroll
    for (int s = 0; s < NSTG - 1; ++s) {
      if (ki < kend) {
        stage_kv8<BK, NT>(p, bh, ki, Ks[ib], Vs[ib], ro, tid);
        ki = advance(ki);
        ib = ib + 1 == NSTG ? 0 : ib + 1;
        ++ahead;
      }
    }
    rope_table();
    wait_vmem_upto<P, NSTG - 1>(ahead);  // the Q loads
    __syncthreads();
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
#pragma unroll
      for (int kk = 0; kk < KK; ++kk) qf[rb][kk] = lds_k8(qs, (rw * RB + rb) * 32 + (lane & 31), kk, lane);
    }
    asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    int cb = 0;
    auto run = [&](auto masked, const int kstop) {
      while (kc < kstop) {
        wait_vmem_upto<P, NSTG - 2>(ahead - 1);  // tile kc has landed
        __syncthreads();
        if (ki < kend) {
          stage_kv8<BK, NT>(p, bh, ki, Ks[ib], Vs[ib], ro, tid);
          ki = advance(ki);
          ib = ib + 1 == NSTG ? 0 : ib + 1;
          ++ahead;
        }
        if (rot && rotate(kc, cb)) __syncthreads();  // rotated keys visible to every wave
        slice(masked, kc, cb);
        --ahead;
        cb = cb + 1 == NSTG ? 0 : cb + 1;
        kc = advance(kc);
      }
    };
    run(std::false_type{}, min(kfull, kend));
    run(std::true_type{}, kend);
  } else {
    int buf = 0;
    if (kc < kend) stage_kv8<BK, NT>(p, bh, kc, Ks[0], Vs[0], ro, tid);
    rope_table();
    wait_vmem();
    __syncthreads();
    if (rot && kc < kend && rotate(kc, 0)) __syncthreads();
    auto run = [&](auto masked, const int kstop) {
      while (kc < kstop) {
        const int kn = advance(kc);
        if (kn < kend) stage_kv8<BK, NT>(p, bh, kn, Ks[buf ^ 1], Vs[buf ^ 1], ro, tid);
        slice(masked, kc, buf);
        wait_vmem();
        __syncthreads();
        if (rot && kn < kend && rotate(kn, buf ^ 1)) __syncthreads();  // the next tile's window rows
        buf ^= 1;
        kc = kn;
      }
    };
    run(std::false_type{}, min(kfull, kend));
    run(std::true_type{}, kend);
  }

  if constexpr (KG > 1) {
    // merge the key groups' (m, l, O) into group 0 through LDS (the stages are
    // free once every wave has passed the barrier):
    // M = max_g m_g, w_g = 2^(m_g - M), O = sum_g w_g O_g, l = sum_g w_g l_g
    constexpr int XO = (KG - 1) * NWR * RB * DB * 16 * 64;
    constexpr int XM = (KG - 1) * NWR * RB * 2 * 64;
    static_assert((XO + XM) * 4 <= (int)sizeof(lds), "exchange fits the K/V stages");
    float* xo = reinterpret_cast<float*>(&lds[0][0][0]);
    float* xm = xo + XO;
    __syncthreads();
    if (kg > 0) {
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) {
        const int slot = ((kg - 1) * NWR + rw) * RB + rb;
#pragma unroll
        for (int db = 0; db < DB; ++db) {
#pragma unroll
          for (int i = 0; i < 16; ++i) xo[((slot * DB + db) * 16 + i) * 64 + lane] = o[rb][db][i];
        }
        xm[(slot * 2) * 64 + lane] = m[rb];
        xm[(slot * 2 + 1) * 64 + lane] = lsum[rb];
      }
    }
    __syncthreads();
    if (kg > 0) return;  // no barrier follows
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      float mg[KG], wg[KG];
      mg[0] = m[rb];
      float M = m[rb];
#pragma unroll
      for (int g = 1; g < KG; ++g) {
        mg[g] = xm[((((g - 1) * NWR + rw) * RB + rb) * 2) * 64 + lane];
        M = fmaxf(M, mg[g]);
      }
#pragma unroll
      for (int g = 0; g < KG; ++g) wg[g] = (mg[g] == -INFINITY) ? 0.f : fast_exp2(mg[g] - M);
      float l = wg[0] * lsum[rb];
#pragma unroll
      for (int g = 1; g < KG; ++g) l += wg[g] * xm[((((g - 1) * NWR + rw) * RB + rb) * 2 + 1) * 64 + lane];
#pragma unroll
      for (int db = 0; db < DB; ++db) {
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          float acc = wg[0] * o[rb][db][i];
#pragma unroll
          for (int g = 1; g < KG; ++g) {
            const int slot = ((g - 1) * NWR + rw) * RB + rb;
            acc += wg[g] * xo[((slot * DB + db) * 16 + i) * 64 + lane];
          }
          o[rb][db][i] = acc;
        }
      }
      m[rb] = M;
      lsum[rb] = l;
    }
  }

#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    lsum[rb] = sum_halves(lsum[rb]);
    if (qrow[rb] >= p.Tq) continue;
    if (nst > 1) {
      // partial of this key range (O already carries the V scale); a split
      // tile's rows are below split_rows
      const long long row = ((long long)split * p.BH + bh) * p.split_rows + qrow[rb];
      float* po = p.part + row * DH;
#pragma unroll
      for (int db = 0; db < DB; ++db) {
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int col = db * 32 + 8 * g + 4 * (lane >> 5);
          f32x4 w;
#pragma unroll
          for (int j = 0; j < 4; ++j) w[j] = o[rb][db][4 * g + j] * p.o_scale;
          *reinterpret_cast<f32x4*>(po + col) = w;
        }
      }
      if (lane < 32) {
        float* ml = p.part + (long long)NS * p.BH * p.split_rows * DH + 2 * row;
        ml[0] = m[rb];
        ml[1] = lsum[rb];
      }
    } else {
      const float inv = p.o_scale / lsum[rb];
      bf16_t* orow = p.o + b_ * p.so.b + h_ * p.so.h + qrow[rb] * p.so.t;
#pragma unroll
      for (int db = 0; db < DB; ++db) {
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int col = db * 32 + 8 * g + 4 * (lane >> 5);
          bf16x4 w;
#pragma unroll
          for (int j = 0; j < 4; ++j) w[j] = to_bf16(o[rb][db][4 * g + j] * inv);
          *reinterpret_cast<bf16x4*>(orow + col) = w;
        }
      }
      if (p.lse != nullptr && lane < 32) {
        p.lse[(long long)bh * p.Tq + qrow[rb]] = (m[rb] + __log2f(lsum[rb])) * 0.69314718055994530942f;
      }
    }
  }
}

// bf16 [B, H, T, D] views -> contiguous e4m3 [B, H, T, D]:
//   code = RNE_e4m3(clamp(fl32(x * inv_scale), -448, 448)).
// One thread per 8 elements; blockIdx.y selects the job (K and V of a commit
// share one launch).
__global__ __launch_bounds__(256) void quantize_fp8_kernel(QuantJobs jobs, int H, int T, int D, long long n_pieces) {
  const QuantJob& jb = jobs.j[blockIdx.y];
  const long long gid = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (gid >= n_pieces) return;
  const int ppr = D / 8;  // pieces per row
  const long long row = gid / ppr;
  const int c = (int)(gid - row * ppr) * 8;
  const long long bh = row / T;
  const long long t = row - bh * T;
  const long long b = bh / H, h = bh - b * H;
  const bf16x8 x = *reinterpret_cast<const bf16x8*>(jb.x + b * jb.sx.b + h * jb.sx.h + t * jb.sx.t + c);
  float f[8];
#pragma unroll
  for (int i = 0; i < 8; ++i) f[i] = fminf(fmaxf((float)x[i] * jb.inv_scale, -kE4m3Max), kE4m3Max);
  u32x2 out;
#pragma unroll
  for (int w = 0; w < 2; ++w) {
    const int lo = __builtin_amdgcn_cvt_pk_fp8_f32(f[4 * w], f[4 * w + 1], 0, false);
    out[w] = (unsigned)__builtin_amdgcn_cvt_pk_fp8_f32(f[4 * w + 2], f[4 * w + 3], lo, true);
  }
  *reinterpret_cast<u32x2*>(jb.y + row * D + c) = out;
}

// Rotation on load of e4m3 window keys (paper Sec. 3.5, re-indexing the
// retained window after an eviction, done when the keys are used rather than
// in place): window chunk blockIdx.y (in window order) is copied from its slot
// to k_win with its rope band rotated by -pend[w] positions.  One thread per
// 128-byte key row; each band pair is decoded, rotated in fp32 with the cos/sin
// of its angle, clamped to +-448 and rounded back to e4m3 (nearest even, the
// quantizer's rounding).  The scale cancels: a rotation is linear, so codes
// are rotated as values.  The cos/sin of pair i are computed once per block,
// in double, as the rotation of one position (cos, sin of its frequency, from
// the host) raised to the power -pend[w] by repeated squaring: no device
// trigonometry, and a relative error of a few 1e-15 for any pend.
__global__ __launch_bounds__(256) void rope_load_fp8_kernel(const fp8_t* __restrict__ k_slots, fp8_t* __restrict__ k_win,
                                                            long long slot_bytes, int S, int first_slot,
                                                            long long pieces, int dim_offset, int n_pairs,
                                                            RopeLoadArgs a) {
  __shared__ float cs[2][64];
  const int w = blockIdx.y;
  if ((int)threadIdx.x < n_pairs) rope_cos_sin(a.pend[w], a.c1[threadIdx.x], a.s1[threadIdx.x], cs[0][threadIdx.x], cs[1][threadIdx.x]);
  __syncthreads();
  // one thread per 16-byte piece (8 pairs) of a key row
  const long long j = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (j >= pieces) return;
  const int slot = first_slot + w < S ? first_slot + w : first_slot + w - S;
  const u32x4 v = *reinterpret_cast<const u32x4*>(k_slots + (long long)slot * slot_bytes + j * 16);
  const int pc = (int)(j % (DH / 16));  // piece of the row
  *reinterpret_cast<u32x4*>(k_win + (long long)w * slot_bytes + j * 16) =
      rope_rotate_piece(v, pc, dim_offset / 2, n_pairs, cs[0], cs[1]);
}

// Tile configuration: 8 waves of one 32-row block (256 queries; one workgroup
// per CU), 128 keys per step.  Measured on the streaming shapes: 128 keys per
// step 12-15% faster than 64; two row blocks per wave (4 waves, one per SIMD)
// 30% slower; 192 keys within 2%.
struct Fwd8Cfg {
  static constexpr int NW = 8;
  static constexpr int RB = 1;
  static constexpr int BN = 128;
  static constexpr int KG = 1;
};

// Few queued rows (a short chunk over a long window) stream the window from
// HBM: 64 rows run 4 waves and 128 rows 8 waves, as 2 key groups of 64 keys
// (128 keys per step, four stages deep), so that every SIMD has a wave at
// work and tiles stay in flight between steps (measured 12% and 6% faster on
// one 64- or 128-token chunk over a 6 x 2640-token window than 2 and 4 waves
// without key groups, double-buffered; 8 waves in 4 groups for 64 rows gain
// nothing more).
template <int NWR>
struct Fwd8FewRows {
  static constexpr int NW = 2 * NWR;
  static constexpr int RB = 1;
  static constexpr int BN = 64;
  static constexpr int KG = 2;
};

template <int NW, int RB, int BN, int KG, bool ROT>
hipError_t launch_fp8_tpl(FwdParams p, const RopeStage& rs, hipStream_t stream) {
  constexpr int BM = 32 * RB * (NW / KG);
  const long long grid = fwd_prepare(p, BM, true);
  hipLaunchKernelGGL((attn_fwd_fp8_kernel<NW, RB, BN, KG, ROT>), dim3((unsigned)grid), dim3(64 * NW), 0, stream, p, rs);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || p.n_splits == 1) return e;
  return launch_combine(p, DH, stream);
}

}  // namespace

// Must agree with the dispatch in launch_fwd_fp8.  Resident workgroups per CU
// from the runtime (fallback one: the few-row configurations hold 128 KB of
// LDS, the 256-row one eight waves of about 230 registers).
FwdChoice fwd8_choice(int Tq) {
  using F2 = Fwd8FewRows<2>;
  using F4 = Fwd8FewRows<4>;
  using C = Fwd8Cfg;
  static const int r64 = resident_workgroups(attn_fwd_fp8_kernel<F2::NW, F2::RB, F2::BN, F2::KG, true>, 64 * F2::NW, 1);
  static const int r128 = resident_workgroups(attn_fwd_fp8_kernel<F4::NW, F4::RB, F4::BN, F4::KG, true>, 64 * F4::NW, 1);
  static const int r256 = resident_workgroups(attn_fwd_fp8_kernel<C::NW, C::RB, C::BN, C::KG, false>, 64 * C::NW, 1);
  if (Tq <= 64) return {64, F2::BN * F2::KG, r64};
  if (Tq <= 128) return {128, F4::BN * F4::KG, r128};
  return {32 * C::RB * C::NW, C::BN, r256};
}

bool fwd8_rotates_in_staging(int Tq, int Tk, int L, const SplitPlan& sp) {
  const FwdChoice ch = fwd8_choice(Tq);
  // with several query tiles per head each key tile is staged once per query
  // tile: those calls rotate the window once, in the separate pass
  if ((Tq + ch.bm - 1) / ch.bm > 1 || L < 1 || Tk < 1) return false;
  if (2 * L < ch.bk) return false;  // a staged tile spans at most three window chunks
  const long long ntiles = (Tk + ch.bk - 1) / ch.bk;
  const long long ns = std::max(sp.n_splits, 1);
  // tiles of one workgroup's key range (whole tiles run every key tile)
  const long long tiles = (sp.n_whole > 0 || ns == 1) ? ntiles : (ntiles + ns - 1) / ns;
  return tiles * ch.bk / L + 2 <= kRopeStageChunks;
}

hipError_t launch_fwd_fp8(FwdParams p, const RopeStage& rs, hipStream_t stream) {
  using F2 = Fwd8FewRows<2>;
  using F4 = Fwd8FewRows<4>;
  using C = Fwd8Cfg;
  const int bm = fwd8_choice(p.Tq).bm;
  if (rs.n_pairs > 0 && (rs.n_pairs > 64 || rs.dim_offset < 0 || rs.dim_offset % 2 != 0 ||
                         rs.dim_offset + 2 * rs.n_pairs > DH))
    return hipErrorInvalidValue;
  if (bm == 64) return launch_fp8_tpl<F2::NW, F2::RB, F2::BN, F2::KG, true>(p, rs, stream);
  if (bm == 128) return launch_fp8_tpl<F4::NW, F4::RB, F4::BN, F4::KG, true>(p, rs, stream);
  // the 256-row configuration without the rotation code unless this call rotates in staging
  if (rs.n_pairs > 0) return launch_fp8_tpl<C::NW, C::RB, C::BN, C::KG, true>(p, rs, stream);
  return launch_fp8_tpl<C::NW, C::RB, C::BN, C::KG, false>(p, rs, stream);
}

hipError_t launch_rope_load_fp8(const uint8_t* k_slots, uint8_t* k_win, long long slot_bytes, int S, int first_slot,
                                int n_window, long long rows_per_slot, int dim_offset, int n_pairs,
                                const RopeLoadArgs& args, hipStream_t stream) {
  const long long pieces = rows_per_slot * (DH / 16);
  if (n_window < 1 || pieces < 1) return hipSuccess;
  if (n_window > 64 || n_pairs < 1 || n_pairs > 64 || pieces > 0x7fffffffLL * 255LL)
    return hipErrorInvalidValue;
  hipLaunchKernelGGL(rope_load_fp8_kernel, dim3((unsigned)((pieces + 255) / 256), (unsigned)n_window), dim3(256), 0,
                     stream, k_slots, k_win, slot_bytes, S, first_slot, pieces, dim_offset, n_pairs, args);
  return hipGetLastError();
}

hipError_t launch_quantize_fp8(const QuantJobs& jobs, int n_jobs, int B, int H, int T, int D, hipStream_t stream) {
  const long long n_pieces = (long long)B * H * T * (D / 8);
  if (n_pieces == 0) return hipSuccess;
  hipLaunchKernelGGL(quantize_fp8_kernel, dim3((unsigned)((n_pieces + 255) / 256), n_jobs), dim3(256), 0, stream,
                     jobs, H, T, D, n_pieces);
  return hipGetLastError();
}

}  // namespace mw
