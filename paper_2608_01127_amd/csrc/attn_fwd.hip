// Block-causal attention forward and cached chunk attention (gfx950).
//
// One workgroup computes 256 query rows of one (batch, head): 4 waves of two
// 32-row blocks at D = 64, 8 waves of one 32-row block at D = 72 and 128
// (FwdCfg).  Cached attention with at most 512 queued rows runs 64- or
// 128-row workgroups whose 8 waves split each key step into key groups
// (FwdDecodeCfg).  Keys are visited in steps of 64 (128 for the key-group
// configurations); each step stages the K and V tile in LDS once for all the
// waves.  Per wave, 32-row block and 32-key block:
//   S^T[key][q] = K Q^T              (bf16 MFMA 32x32x16, fp32 accumulate;
//                                     Q stays in registers as the B operand)
//   online softmax over keys         (a query is one lane column of S^T, so
//                                     the row max/sum are in-lane reductions
//                                     plus one exchange with lane l^32)
//   O^T[d][q] += V^T P^T             (P^T feeds the MFMA B operand from the
//                                     accumulator registers; V^T is read from
//                                     the row-major V tile with transposing
//                                     LDS reads)
// Key steps wholly above the chunk diagonal are never visited; steps wholly
// below it skip the mask; only steps that straddle a chunk edge (or the end of
// the keys) evaluate it per element.
//
// Visibility rule: paper Sec. 3.2 (block-causal chunks) for training and
// Sec. 3.5 (queued in-flight chunks over committed history) for the cached
// variant; see Vis in mw_device.h.
#include <algorithm>
#include <cmath>
#include <map>
#include <mutex>
#include <queue>
#include <tuple>
#include <vector>
#include <type_traits>

#include "mw_device.h"
#include "mw_kernels.h"

namespace mw {

// Per-thread row offsets of the K and V tiles: queued / training keys (their
// views' T strides) and ring slots (rows D apart).
template <int D, bool CACHED, int BN, int NT>
struct KVOffsets {
  RowOffsets<D, BN, NT> k, v, w;
  __device__ __forceinline__ KVOffsets(const FwdParams& p, int tid)
      : k(p.sk.t, tid), v(p.sv.t, tid), w(CACHED ? D : 0, tid) {}
};

// Staging of one K/V tile straight into LDS.  Key rows past the end of the
// (virtual) key sequence read the last key instead; the mask hides them.
// A tile of equally spaced rows (almost every tile) is staged from one
// wave-uniform base pointer plus the per-thread offsets above.  Cached
// attention: the key sequence is the sink, then the window chunks in ring
// slots, then the queued chunks; a tile inside one window chunk or inside the
// queued keys is recognised with scalar tests, and only tiles that straddle a
// boundary (or the ragged end) take the per-row mapping.
template <int D, bool CACHED, int BN, int NT>
__device__ __forceinline__ void stage_kv(const FwdParams& p, int bh, long long kbase, long long vbase, int k0,
                                         bf16_t* Kt, bf16_t* Vt, const KVOffsets<D, CACHED, BN, NT>& ro, int tid) {
  const long long skt = p.sk.t, svt = p.sv.t;
  if constexpr (CACHED) {
    const int kl = min(k0 + BN, p.Tk) - 1;  // last real key of the tile
    const int kw0 = k0 - p.sink_len;
    const int w0 = kw0 > 0 ? kw0 / p.L : 0;
    const int off0 = kw0 - w0 * p.L;
    if (k0 >= p.wL && k0 + BN <= p.Tk) {  // queued keys only, a whole tile
      const long long j = k0 - p.wL;
      stage_rows_s<D, BN, NT>(Kt, p.k + kbase + j * skt, ro.k, tid);
      stage_rows_s<D, BN, NT>(Vt, p.v + vbase + j * svt, ro.v, tid);
      return;
    }
    if (kw0 >= 0 && kl < p.wL && off0 + (kl - k0) < p.L) {  // one window chunk
      int slot = p.first_slot + w0;
      slot = slot >= p.S ? slot - p.S : slot;
      const long long e = (long long)slot * p.slot_stride + ((long long)bh * p.L + off0) * D;
      stage_rows_s<D, BN, NT>(Kt, p.k_slots + e, ro.w, tid);
      stage_rows_s<D, BN, NT>(Vt, p.v_slots + e, ro.w, tid);
      return;
    }
    // a tile straddling the sink, chunk or queued boundaries, or the end:
    // row by row (the window chunk of the first key is found once; a row
    // moves on by whole chunks from there)
    stage_kv_rows_direct<D, BN, NT>(Kt, Vt, [&](int r) -> RowPair {
      const int key = min(k0 + r, p.Tk - 1);
      if (key < p.sink_len) {
        const long long e = ((long long)bh * p.sink_len + key) * D;
        return {p.k_sink + e, p.v_sink + e};
      }
      if (key < p.wL) {
        int w = w0, off = key - p.sink_len - w0 * p.L;
        while (off >= p.L) {  // at most one step when L >= BN
          off -= p.L;
          ++w;
        }
        int slot = p.first_slot + w;
        slot = slot >= p.S ? slot - p.S : slot;
        const long long e = (long long)slot * p.slot_stride + ((long long)bh * p.L + off) * D;
        return {p.k_slots + e, p.v_slots + e};
      }
      const long long j = key - p.wL;
      return {p.k + kbase + j * skt, p.v + vbase + j * svt};
    }, tid);
  } else {
    if (k0 + BN <= p.Tk) {
      stage_rows_s<D, BN, NT>(Kt, p.k + kbase + (long long)k0 * skt, ro.k, tid);
      stage_rows_s<D, BN, NT>(Vt, p.v + vbase + (long long)k0 * svt, ro.v, tid);
      return;
    }
    stage_kv_rows_direct<D, BN, NT>(Kt, Vt, [&](int r) -> RowPair {  // the ragged last tile
      const long long j = min(k0 + r, p.Tk - 1);
      return {p.k + kbase + j * skt, p.v + vbase + j * svt};
    }, tid);
  }
}

// Rows of the running max only move when a tile raises it by more than this
// many powers of two; until then probabilities are taken against the stale
// max (they stay below 2^8, far from fp32/bf16 limits).  The normaliser uses
// the same reference, so the result is unchanged up to rounding, and the
// O rescale is skipped on almost every step.
constexpr float kRescaleThreshold = 8.f;

// K/V stages of a configuration: two (double buffering) except for the
// four-wave key-group configuration of 64 queued rows, which streams 64-key
// tiles four deep.
constexpr int fwd_stages(int nw, int kg) { return kg > 1 && nw == 4 ? 4 : 2; }

// NW waves per workgroup, each owning RB blocks of 32 query rows; BN keys per
// main-loop step.  With RB = 2 every K and V fragment read from LDS feeds two
// MFMAs (one per row block), halving LDS traffic per MFMA: with one 32-row
// block per wave the LDS bandwidth (128 B/clk/CU) equals what four waves
// consume at the full MFMA rate.
// KG key groups: the NW waves form KG groups of NW / KG waves; a step stages
// KG * BN keys and group g works on its BN-key slice, so KG groups cover
// different keys of the same query rows and merge (m, l, O) through LDS at
// the end.  With few query rows this keeps all four SIMDs of a CU busy.
template <int D, bool CACHED, int NW, int BN, int RB, int KG>
__global__ __launch_bounds__(64 * NW, (8 / NW) > 0 ? (8 / NW) : 1) void attn_fwd_kernel(FwdParams p) {
  static_assert(NW % KG == 0, "waves split evenly into key groups");
  constexpr int NWR = NW / KG;           // waves per key group (row waves)
  constexpr int BM = 32 * RB * NWR, NT = 64 * NW, KB = BN / 32;
  constexpr int BK = BN * KG;            // keys staged per step
  constexpr int KK = (D + 15) / 16;  // contraction steps over D (D = 72: the last one half zeros)
  constexpr int DB = (D + 31) / 32;  // 32-wide column blocks of D (D = 72: the last one 8 wide)
  constexpr int TE = stage_elems<D, BK, NT>();  // elements of one staged tile buffer
  constexpr int NSTG = fwd_stages(NW, KG);      // K/V stages (see the main loop)
  __shared__ __attribute__((aligned(16))) bf16_t lds[2][NSTG][TE];  // K, V x stages
  bf16_t(*Ks)[TE] = lds[0];
  bf16_t(*Vs)[TE] = lds[1];

  const int NS = p.n_splits;  // key ranges of a split tile (partials layout)
  int bh, qt, split, nst;      // nst: key ranges of this workgroup's tile
  if constexpr (CACHED) {
    cached_item(blockIdx.x, gridDim.x, p.n_qtiles, NS, p.n_whole, bh, qt, split, nst);
  } else {
    fwd_item(blockIdx.x, gridDim.x, p.BH, p.n_qtiles, NS, bh, qt, split);
    nst = NS;
  }
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int rw = wave % NWR, kg = wave / NWR;  // row wave, key group
  const int q0 = qt * BM;
  const int b_ = bh / p.H, h_ = bh - b_ * p.H;
  const long long qbase = b_ * p.sq.b + h_ * p.sq.h;
  const long long kbase = b_ * p.sk.b + h_ * p.sk.h;
  const long long vbase = b_ * p.sv.b + h_ * p.sv.h;

  Vis vis{p.vis_mode, p.L, p.Tk, p.qlen, p.wL};

  // Per row block: this lane's query row, its Q fragments (B operand of
  // S^T = K Q^T: Q[qrow][16kk + 8(l/32) + 0..7]) and its visible key ranges.
  int qrow[RB], e1[RB], s2[RB], e2[RB];
  bf16x8 qf[RB][KK];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    qrow[rb] = q0 + (rw * RB + rb) * 32 + (lane & 31);
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
      if constexpr (NSTG > 2) break;  // staged through LDS with the first K/V tiles
      if (qrow[rb] < p.Tq && (D % 16 == 0 || 16 * kk + 8 * (lane >> 5) < D)) {
        qf[rb][kk] = *reinterpret_cast<const bf16x8*>(p.q + qbase + qrow[rb] * p.sq.t + 16 * kk + 8 * (lane >> 5));
      } else {  // rows past Tq and columns past D contribute zeros
#pragma unroll
        for (int j = 0; j < 8; ++j) qf[rb][kk][j] = (__bf16)0.f;
      }
    }
    vis.range(min(qrow[rb], p.Tq - 1), e1[rb], s2[rb], e2[rb]);
  }
  int e1f, s2f, e2f, e1l, s2l, e2l;
  vis.range(q0, e1f, s2f, e2f);
  vis.range(min(q0 + BM, p.Tq) - 1, e1l, s2l, e2l);
  const int kend_all = max(e1l, e2l);
  // this workgroup's share of the key tiles [0, kend_all): split `split` of nst
  const int ntiles = (kend_all + BK - 1) / BK;
  const int kbeg = (int)((long long)ntiles * split / nst) * BK;
  const int kend = min(kend_all, (int)((long long)ntiles * (split + 1) / nst) * BK);
  // next visited key tile after k: tiles no row of this workgroup can see are skipped
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
  const float c = p.scale_log2;

  // Tiles [0, kfull) are visible to every row of the workgroup and run without
  // any mask code; the remaining tiles (chunk edges, the ragged end, the gap of
  // the isolated rule) run the masked instantiation.  Separate loops keep the
  // fast loop free of the mask and of register copies between the two bodies.
  const int kfull = max(0, (e1f / BK) * BK);

  // Per-lane element offsets, within a staged tile, of this wave's fragment
  // reads: the K rows of S^T = K Q^T (one per 16-column contraction step) and
  // the two transposing reads of each 32-column block of V.  The tile swizzle
  // repeats every 16 rows, so a 32-key block or a 16-key contraction step only
  // adds a constant: a fragment address is the stage buffer plus one of these
  // registers (one add, shared by the key blocks) plus an immediate.  A key
  // group's slice of the staged keys is folded in here.
  const FragOffsets<D> fo(lane, kg * BN * D);

  auto step = [&](auto masked, const int k0, const bf16_t* Kt, const bf16_t* Vt) {
    // S^T for KB 32-key blocks x RB row blocks; each K fragment is read once
    f32x16 s[RB][KB];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb)
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) s[rb][kb] = zero16();
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) {
        const bf16x8 kfrag = fo.row8(Kt, kb * 32, kk);
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) s[rb][kb] = mfma32(kfrag, qf[rb][kk], s[rb][kb]);
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
            // non-short-circuit form: evaluated as compares and one select, without
            // branches (a branchy lowering of the short-circuit form clobbered the
            // accumulator element before the second range was tested)
            const bool ok = (key < e1[rb]) | ((key >= s2[rb]) & (key < e2[rb]));
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
      mx[rb] = max_halves(mx[rb]) * c;  // scaled row max of this tile (log2 units)
      need[rb] = mx[rb] > m[rb] + kRescaleThreshold;
      need_any |= need[rb];
    }
    if (wave_any(need_any)) {
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) {
        // lanes that move their max rescale by 2^(m - mx) (0 while m is still -inf);
        // the others keep alpha = 1 (their m may still be -inf: no -inf - -inf)
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
          ls += pv;
        }
      }
      lsum[rb] += ls;
    }

    // O^T += V^T P^T; each V fragment is read once for all row blocks
#pragma unroll
    for (int kb = 0; kb < KB; ++kb) {
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        bf16x8 pb[RB];
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) pb[rb] = pack8(s[rb][kb], t);
#pragma unroll
        for (int db = 0; db < DB; ++db) {
          const bf16x8 vfrag = fo.tr8(Vt, kb * 32, t, db);
#pragma unroll
          for (int rb = 0; rb < RB; ++rb) o[rb][db] = mfma32(vfrag, pb[rb], o[rb][db]);
        }
      }
    }
  };

  // this wave's slice of a staged step: keys [kg * BN, (kg + 1) * BN)
  auto slice = [&](auto masked, const int k0, const int st) { step(masked, k0 + kg * BN, Ks[st], Vs[st]); };
  const KVOffsets<D, CACHED, BK, NT> kvo(p, tid);
  int kc = advance(kbeg - BK);  // next tile to use
  if constexpr (NSTG > 2) {
    // Streaming configurations (few query rows, bound by reading the keys):
    // up to NSTG - 1 tiles in flight.  Each wave waits only for the oldest of
    // its outstanding tiles (s_waitcnt on the vector-memory counter, which the
    // LDS-direct loads of a tile decrement in issue order), then one barrier
    // makes the tile visible and frees the buffer computed last, which takes
    // the next tile.  A tile is 2 * ROUNDS loads per thread on every path.
    // The Q tile is staged the same way, first, into the last stage buffer
    // (64 rows in its K half, the next 64 in its V half), which the first
    // tiles leave free; every Q load has landed once at most the tiles' loads
    // are outstanding, and the Q fragments are read from LDS before the first
    // barrier of the loop frees that buffer.  (Loading Q straight into
    // registers would leave the compiler, which cannot see the LDS-direct
    // loads, waiting for all outstanding loads inside the loop.)
    constexpr int P = 2 * StagePlan<D, BK, NT>::ROUNDS;
    static_assert(P * (NSTG - 1) <= 63, "vector-memory counter range");
    static_assert(BM % 64 == 0 && BM <= 128 && TE >= 64 * D, "the Q tile fits the last stage buffer");
#pragma unroll
    for (int h = 0; h < BM / 64; ++h) {
      bf16_t* qs = h == 0 ? Ks[NSTG - 1] : Vs[NSTG - 1];
      stage_rows_direct<D, 64, NT>(qs, [&](int r) { return p.q + qbase + min(q0 + 64 * h + r, p.Tq - 1) * p.sq.t; },
                                   tid);
    }
    int ki = kc, ib = 0, ahead = 0;  // next tile to issue, its buffer, tiles issued and not yet used
#pragma unroll
    for (int s = 0; s < NSTG - 1; ++s) {
      if (ki < kend) {
        stage_kv<D, CACHED, BK, NT>(p, bh, kbase, vbase, ki, Ks[ib], Vs[ib], kvo, tid);
        ki = advance(ki);
        ib = ib + 1 == NSTG ? 0 : ib + 1;
        ++ahead;
      }
    }
    wait_vmem_upto<P, NSTG - 1>(ahead);  // the Q loads
    __syncthreads();
    {
      const FragOffsets<D> fq(lane, 0);
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) {
        const int r0 = (rw * RB + rb) * 32;  // this row block within the Q tile
        const bf16_t* qs = r0 < 64 ? Ks[NSTG - 1] : Vs[NSTG - 1];
#pragma unroll
        for (int kk = 0; kk < KK; ++kk) qf[rb][kk] = fq.row8(qs, r0 & 63, kk);
      }
      asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    }
    int cb = 0;
    auto run = [&](auto masked, const int kstop) {
      while (kc < kstop) {
        wait_vmem_upto<P, NSTG - 2>(ahead - 1);  // tile kc has landed
        __syncthreads();
        if (ki < kend) {
          stage_kv<D, CACHED, BK, NT>(p, bh, kbase, vbase, ki, Ks[ib], Vs[ib], kvo, tid);
          ki = advance(ki);
          ib = ib + 1 == NSTG ? 0 : ib + 1;
          ++ahead;
        }
        slice(masked, kc, cb);
        --ahead;
        cb = cb + 1 == NSTG ? 0 : cb + 1;
        kc = advance(kc);
      }
    };
    run(std::false_type{}, min(kfull, kend));
    run(std::true_type{}, kend);
  } else {
    // double buffering: the next tile streams in during this step's math
    int buf = 0;
    if (kc < kend) stage_kv<D, CACHED, BK, NT>(p, bh, kbase, vbase, kc, Ks[0], Vs[0], kvo, tid);
    wait_vmem();
    __syncthreads();
    auto run = [&](auto masked, const int kstop) {
      while (kc < kstop) {
        const int kn = advance(kc);
        if (kn < kend) stage_kv<D, CACHED, BK, NT>(p, bh, kbase, vbase, kn, Ks[buf ^ 1], Vs[buf ^ 1], kvo, tid);
        slice(masked, kc, buf);
        wait_vmem();
        __syncthreads();
        buf ^= 1;
        kc = kn;
      }
    };
    run(std::false_type{}, min(kfull, kend));
    run(std::true_type{}, kend);
  }

  if constexpr (KG > 1) {
    // Merge the key groups' partial results into group 0 through LDS (the K/V
    // stages are free once every wave has passed this barrier):
    // M = max_g m_g, w_g = 2^(m_g - M), O = sum_g w_g O_g, l = sum_g w_g l_g.
    constexpr int XO = (KG - 1) * NWR * RB * DB * 16 * 64;  // floats of O
    constexpr int XM = (KG - 1) * NWR * RB * 2 * 64;        // floats of (m, l)
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
        const int slot = ((g - 1) * NWR + rw) * RB + rb;
        mg[g] = xm[(slot * 2) * 64 + lane];
        M = fmaxf(M, mg[g]);
      }
#pragma unroll
      for (int g = 0; g < KG; ++g) wg[g] = (mg[g] == -INFINITY) ? 0.f : fast_exp2(mg[g] - M);
      float l = wg[0] * lsum[rb];
#pragma unroll
      for (int g = 1; g < KG; ++g) {
        const int slot = ((g - 1) * NWR + rw) * RB + rb;
        l += wg[g] * xm[(slot * 2 + 1) * 64 + lane];
      }
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
      // partial result of this key range: unnormalised O, the reference max m
      // (log2 units, possibly stale by up to the rescale threshold) and the sum
      // l of 2^(s - m); rows past Tq are not written (a split tile's rows are
      // below split_rows)
      const long long row = ((long long)split * p.BH + bh) * p.split_rows + qrow[rb];
      float* po = p.part + row * D;
#pragma unroll
      for (int db = 0; db < DB; ++db) {
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int col = db * 32 + 8 * g + 4 * (lane >> 5);
          if (D % 32 != 0 && col >= D) continue;  // (D = 72)
          f32x4 w;
#pragma unroll
          for (int j = 0; j < 4; ++j) w[j] = o[rb][db][4 * g + j];
          *reinterpret_cast<f32x4*>(po + col) = w;
        }
      }
      if (lane < 32) {
        float* ml = p.part + (long long)NS * p.BH * p.split_rows * D + 2 * row;
        ml[0] = m[rb];
        ml[1] = lsum[rb];
      }
    } else {
      const float inv = 1.f / lsum[rb];
      bf16_t* orow = p.o + b_ * p.so.b + h_ * p.so.h + qrow[rb] * p.so.t;
#pragma unroll
      for (int db = 0; db < DB; ++db) {
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int col = db * 32 + 8 * g + 4 * (lane >> 5);
          if (D % 32 != 0 && col >= D) continue;  // (D = 72)
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

// Tile configuration per head dimension: waves per workgroup (32 query rows
// each), keys per step, row blocks per wave and LDS stages.  With D = 128 a
// workgroup of 8 waves shares each staged K/V tile among 256 queries, halving
// L2 -> LDS traffic per MFMA; with D = 64 four waves of two row blocks (two
// workgroups per CU) measured faster.
template <int D>
struct FwdCfg {
  static constexpr int NW = D == 64 ? 4 : 8;
  static constexpr int BN = 64;
  static constexpr int RB = D == 64 ? 2 : 1;  // 32-row query blocks per wave
  static constexpr int KG = 1;
};
// (D = 72, the 0.5B model's head width, runs the D = 128 arrangement: its
// wider accumulators leave no room for two row blocks per wave.)

// Cached attention with few queued rows (a short chunk over a long window) is
// bound by streaming the window from HBM.  The waves split into key groups of
// row waves: for 64 rows, four waves in 2 groups of 2 stage 64 keys per step,
// four stages deep (one wave per SIMD; measured 3-4% faster than eight waves
// in 4 groups double-buffering 128-key steps, whose bulk waits leave the
// memory pipe idle between steps); for 128 rows, eight waves in 2 groups of 4
// stage 128 keys per step, double-buffered.
// Up to 512 queued rows run as 128-row tiles of this kind (their workgroups read
// the same window, which the L2 and the Infinity Cache share): measured 20% and
// 11% faster than 256-row tiles at 256 and 512 rows over a 6 x 2640-token window.
template <int D, int NWR>
struct FwdDecodeCfg {
  static constexpr int NW = NWR == 2 ? 4 : 8;
  static constexpr int KG = NW / NWR;
  static constexpr int BN = NWR == 2 ? 32 : 128 / KG;
  static constexpr int RB = 1;
};

// Merge of the per-split partials: with M = max_s m_s and w_s = 2^(m_s - M),
//   O = sum_s w_s O_s / sum_s w_s l_s,   LSE = (M + log2 sum_s w_s l_s) ln 2.
// The split rows are rows [0, split_rows) of each head (rows = BH * split_rows).
// One thread per 4 output columns of a row.
template <int D, int G>
__global__ __launch_bounds__(256) void attn_combine_kernel(const float* __restrict__ part, uint16_t* __restrict__ o,
                                                           Strides so, int H, int Tq, int split_rows,
                                                           float* __restrict__ lse, int NS, long long rows) {
  constexpr int TPR = D / 4;  // threads per row
  const long long gid = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  const long long row = gid / TPR;
  if (row >= rows) return;
  const long long bh = row / split_rows;
  const long long t = row - bh * split_rows;
  const long long orow = (bh / H) * so.b + (bh % H) * so.h + t * so.t;
  const int c = (int)(gid % TPR) * 4;
  const float* ml = part + (long long)NS * rows * D;
  // One pass over the splits, G at a time with all their loads in flight (one
  // round trip for up to G splits; G is the smallest of 4, 8, 16 that covers
  // the split count, or 16): a running reference M, rescaled when a group
  // raises it, as in the attention kernel itself.
  float M = -INFINITY, L = 0.f;
  f32x4 acc = {0.f, 0.f, 0.f, 0.f};
  for (int s0 = 0; s0 < NS; s0 += G) {
    float mv[G], lv[G];
    f32x4 v[G];
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const long long r = (long long)(s0 + g) * rows + row;
      const bool in = s0 + g < NS;
      mv[g] = in ? ml[2 * r] : -INFINITY;
      lv[g] = in ? ml[2 * r + 1] : 0.f;
      v[g] = in ? *reinterpret_cast<const f32x4*>(part + r * D + c) : f32x4{0.f, 0.f, 0.f, 0.f};
    }
    float Mn = M;
#pragma unroll
    for (int g = 0; g < G; ++g) Mn = fmaxf(Mn, mv[g]);
    if (Mn == -INFINITY) continue;  // no keys in these splits (or so far)
    const float a = (M == -INFINITY) ? 0.f : fast_exp2(M - Mn);
    L *= a;
#pragma unroll
    for (int j = 0; j < 4; ++j) acc[j] *= a;
#pragma unroll
    for (int g = 0; g < G; ++g) {
      const float w = (mv[g] == -INFINITY) ? 0.f : fast_exp2(mv[g] - Mn);  // empty split: no keys
      L = fmaf(w, lv[g], L);
#pragma unroll
      for (int j = 0; j < 4; ++j) acc[j] = fmaf(w, v[g][j], acc[j]);
    }
    M = Mn;
  }
  const float inv = 1.f / L;
  bf16x4 out;
#pragma unroll
  for (int j = 0; j < 4; ++j) out[j] = to_bf16(acc[j] * inv);
  *reinterpret_cast<bf16x4*>(o + orow + c) = out;
  if (lse != nullptr && c == 0) lse[bh * Tq + t] = (M + __log2f(L)) * 0.69314718055994530942f;
}

// The merge kernel for p's split rows, with its group size chosen by the split count.
template <int D>
static hipError_t launch_combine_d(const FwdParams& p, hipStream_t stream) {
  const long long rows = (long long)p.BH * p.split_rows;
  const long long threads = rows * (D / 4);
  const dim3 grid((unsigned)((threads + 255) / 256));
  if (p.n_splits <= 4) {
    hipLaunchKernelGGL((attn_combine_kernel<D, 4>), grid, dim3(256), 0, stream, p.part, p.o, p.so, p.H, p.Tq,
                       p.split_rows, p.lse, p.n_splits, rows);
  } else if (p.n_splits <= 8) {
    hipLaunchKernelGGL((attn_combine_kernel<D, 8>), grid, dim3(256), 0, stream, p.part, p.o, p.so, p.H, p.Tq,
                       p.split_rows, p.lse, p.n_splits, rows);
  } else {
    hipLaunchKernelGGL((attn_combine_kernel<D, 16>), grid, dim3(256), 0, stream, p.part, p.o, p.so, p.H, p.Tq,
                       p.split_rows, p.lse, p.n_splits, rows);
  }
  return hipGetLastError();
}

template <int D, bool CACHED, int NW, int BN, int RB, int KG>
static hipError_t launch_fwd_tpl(FwdParams p, hipStream_t stream) {
  constexpr int BM = 32 * RB * (NW / KG);
  const long long grid = fwd_prepare(p, BM, CACHED);
  hipLaunchKernelGGL((attn_fwd_kernel<D, CACHED, NW, BN, RB, KG>), dim3((unsigned)grid), dim3(64 * NW), 0, stream, p);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || p.n_splits == 1) return e;
  return launch_combine_d<D>(p, stream);
}

template <int D, bool CACHED>
static hipError_t launch_fwd_cfg(const FwdParams& p, hipStream_t stream) {
  using C = FwdCfg<D>;
  return launch_fwd_tpl<D, CACHED, C::NW, C::BN, C::RB, C::KG>(p, stream);
}

// This file is compiled once per head dimension (MW_FWD_HEAD_DIM = 64, 72 or 128),
// with the instruction-scheduling option measured faster for each; the merge
// kernel and the split planner live in the D = 128 unit.  Two D = 128 cached
// configurations are compiled in units of their own: the 256-row one
// (MW_FWD_CACHED) with 64-byte loop alignment (measured 2-4% faster on the
// cached calls, and 1.7% slower on the training kernel, which therefore stays
// in the main unit), and the key-group configurations for few queued rows
// (MW_FWD_DECODE) with the default scheduler.
template <int D, bool CACHED, int NW, int BN, int RB, int KG>
static int resident_tpl(int fallback) {
  static const int n = resident_workgroups(attn_fwd_kernel<D, CACHED, NW, BN, RB, KG>, 64 * NW, fallback);
  return n;
}

template <int D, bool CACHED>
static int resident_cfg(int fallback) {
  using C = FwdCfg<D>;
  return resident_tpl<D, CACHED, C::NW, C::BN, C::RB, C::KG>(fallback);
}

// (fallbacks: D = 64 runs 4 waves of about 235 registers, two workgroups per
// CU; D = 72 and 128 run 8 waves of 160-240 registers, one per CU)
#if MW_FWD_HEAD_DIM == 64 && !defined(MW_FWD_DECODE)
hipError_t launch_fwd_64(const FwdParams& p, bool cached, hipStream_t stream) {
  return cached ? launch_fwd_cfg<64, true>(p, stream) : launch_fwd_cfg<64, false>(p, stream);
}
int fwd_resident_wgs_64(bool cached) { return cached ? resident_cfg<64, true>(2) : resident_cfg<64, false>(2); }
#elif MW_FWD_HEAD_DIM == 72 && !defined(MW_FWD_DECODE)
hipError_t launch_fwd_72(const FwdParams& p, bool cached, hipStream_t stream) {
  return cached ? launch_fwd_cfg<72, true>(p, stream) : launch_fwd_cfg<72, false>(p, stream);
}
int fwd_resident_wgs_72(bool cached) { return cached ? resident_cfg<72, true>(1) : resident_cfg<72, false>(1); }
#elif MW_FWD_HEAD_DIM == 128 && !defined(MW_FWD_DECODE) && !defined(MW_FWD_CACHED)
int fwd_resident_wgs_128(bool cached) { return cached ? fwd_resident_wgs_cached_128() : resident_cfg<128, false>(1); }
hipError_t launch_fwd_128(const FwdParams& p, bool cached, hipStream_t stream) {
  if (!cached) return launch_fwd_cfg<128, false>(p, stream);
  const int bm = fwd_choice(128, true, p.Tq).bm;
  if (bm != 32 * FwdCfg<128>::RB * FwdCfg<128>::NW) return launch_fwd_decode_128(p, bm, stream);
  return launch_fwd_cached_128(p, stream);
}
#elif MW_FWD_HEAD_DIM == 128 && defined(MW_FWD_CACHED)
hipError_t launch_fwd_cached_128(const FwdParams& p, hipStream_t stream) {
  return launch_fwd_cfg<128, true>(p, stream);
}
int fwd_resident_wgs_cached_128() { return resident_cfg<128, true>(1); }
#elif MW_FWD_HEAD_DIM == 128 && defined(MW_FWD_DECODE)
hipError_t launch_fwd_decode_128(const FwdParams& p, int bm, hipStream_t stream) {
  if (bm == 64) {
    using C = FwdDecodeCfg<128, 2>;
    return launch_fwd_tpl<128, true, C::NW, C::BN, C::RB, C::KG>(p, stream);
  }
  using C = FwdDecodeCfg<128, 4>;
  return launch_fwd_tpl<128, true, C::NW, C::BN, C::RB, C::KG>(p, stream);
}
// (fallback: 4 or 8 waves of 180-245 registers and 128 KB of LDS, one per CU)
int fwd_resident_wgs_decode_128(int bm) {
  using C2 = FwdDecodeCfg<128, 2>;
  using C4 = FwdDecodeCfg<128, 4>;
  return bm == 64 ? resident_tpl<128, true, C2::NW, C2::BN, C2::RB, C2::KG>(1)
                  : resident_tpl<128, true, C4::NW, C4::BN, C4::RB, C4::KG>(1);
}
#else
#error "compile with -DMW_FWD_HEAD_DIM=64, 72 or 128 (128 optionally with -DMW_FWD_CACHED or -DMW_FWD_DECODE)"
#endif

#if MW_FWD_HEAD_DIM == 128 && !defined(MW_FWD_DECODE) && !defined(MW_FWD_CACHED)
// Must agree with the dispatch in launch_fwd_128.
FwdChoice fwd_choice(int D, bool cached, int Tq) {
  using C2 = FwdDecodeCfg<128, 2>;
  using C4 = FwdDecodeCfg<128, 4>;
  if (cached && D == 128 && Tq <= 64) return {64, C2::BN * C2::KG, fwd_resident_wgs_decode_128(64)};
  if (cached && D == 128 && Tq <= 512)  // 128-row tiles up to 512 rows
    return {128, C4::BN * C4::KG, fwd_resident_wgs_decode_128(128)};
  if (D == 64) return {32 * FwdCfg<64>::RB * FwdCfg<64>::NW, FwdCfg<64>::BN, fwd_resident_wgs_64(cached)};
  if (D == 72) return {32 * FwdCfg<72>::RB * FwdCfg<72>::NW, FwdCfg<72>::BN, fwd_resident_wgs_72(cached)};
  return {32 * FwdCfg<128>::RB * FwdCfg<128>::NW, FwdCfg<128>::BN, fwd_resident_wgs_128(cached)};
}

hipError_t launch_combine(const FwdParams& p, int D, hipStream_t stream) {
  if (D != 128) return hipErrorInvalidValue;
  return launch_combine_d<128>(p, stream);
}

size_t fwd_split_bytes(int D, int BH, int split_rows, int n_splits) {
  if (n_splits <= 1) return 0;
  return (size_t)n_splits * BH * split_rows * (D + 2) * sizeof(float);
}

int fwd_split_rows(int bm, int Tq, const SplitPlan& sp) {
  if (sp.n_splits <= 1) return 0;
  const int nqt = (Tq + bm - 1) / bm;
  return std::min(Tq, (nqt - std::min(std::max(sp.n_whole, 0), nqt)) * bm);
}

// Sustained MFMA rate of the bf16 cached kernel assumed by the split planner.
constexpr double kBf16Flops = 1.1e15;

SplitPlan fwd_plan_cached(int D, int BH, int Tq, int Tk, int qlen, bool isolated, size_t ws_bytes) {
  return fwd_plan_splits(fwd_choice(D, true, Tq), kBf16Flops, 2, D, BH, Tq, Tk, qlen, isolated, ws_bytes);
}

namespace {

// Makespan, in key steps, of the cached grid's workgroups on `slots` resident
// workgroup slots, taken in dispatch order (cached_item) each as soon as a
// slot frees: `heads` heads of query tiles with steps[qt] key steps each, the
// n_whole heaviest unsplit, the rest over ns key ranges.  A workgroup costs
// its key steps plus `o_wg`, plus `o_part` when it writes a partial.
double split_makespan(const std::vector<int>& steps, int heads, int slots, int ns, int n_whole, double o_wg,
                      double o_part) {
  std::priority_queue<double, std::vector<double>, std::greater<double>> free_at;
  for (int i = 0; i < slots; ++i) free_at.push(0.0);
  auto take = [&](double t) {
    const double s = free_at.top();
    free_at.pop();
    free_at.push(s + t);
  };
  const int nqt = (int)steps.size();
  for (int h = 0; h < heads; ++h) {
    for (int r = 0; r < n_whole; ++r) take(steps[nqt - 1 - r] + o_wg);
    for (int s = 0; s < ns; ++s) {
      for (int r = n_whole; r < nqt; ++r) {
        const long long c = steps[nqt - 1 - r];
        take((double)(c * (s + 1) / ns - c * s / ns) + o_wg + o_part);
      }
    }
  }
  double mk = 0.0;
  while (!free_at.empty()) {
    mk = std::max(mk, free_at.top());
    free_at.pop();
  }
  return mk;
}

struct PlanKey {
  int bm, bk, wg, kv_bytes, D, BH, Tq, Tk, qlen, isolated;
  double flops;
  size_t ws;
  bool operator<(const PlanKey& o) const {
    return std::tie(bm, bk, wg, kv_bytes, D, BH, Tq, Tk, qlen, isolated, flops, ws) <
           std::tie(o.bm, o.bk, o.wg, o.kv_bytes, o.D, o.BH, o.Tq, o.Tk, o.qlen, o.isolated, o.flops, o.ws);
  }
};

SplitPlan plan_splits(const FwdChoice& ch, double flops, int kv_bytes, int D, int BH, int Tq, int Tk, int qlen,
                      bool isolated, size_t ws_bytes) {
  const double cus = 256.0;
  const double slots = cus * ch.wg_per_cu;
  const int nqt = (Tq + ch.bm - 1) / ch.bm;
  const double base = (double)nqt * BH;
  const double pairs = (double)BH * Tq * std::max(1.0, (double)Tk - 0.5 * Tq);
  const double t_mfma = 4.0 * pairs * D / flops;
  const double t_stream = 2.0 * BH * (double)Tk * D * kv_bytes / 4.0e12;
  const int ns_max = (int)std::min<long long>(64, std::max(1, (Tk / 128) / 2));
  auto part_time = [&](int rows, int ns) { return ns > 1 ? 2.0 * fwd_split_bytes(D, BH, rows, ns) / 4.0e12 : 0.0; };
  struct Cand {
    double t;
    SplitPlan sp;
  };
  std::vector<Cand> cands;
  if (t_mfma < t_stream) {
    // streaming-bound (few query rows): every tile split, priced by CU coverage
    for (int ns = 1; ns <= ns_max; ++ns) {
      if (ns > 1 && fwd_split_bytes(D, BH, Tq, ns) > ws_bytes) break;
      cands.push_back({t_stream / std::min(1.0, base * ns / cus) + part_time(Tq, ns), {ns, 0}});
    }
  } else if (base >= 8.0 * slots) {
    // eight or more rounds of workgroups: the last round is a small fraction
    // of the call, so nothing is split
    cands.push_back({t_mfma, {1, 0}});
  } else {
    // MFMA-bound: simulate the dispatch of one XCD (BH / 8 whole heads when
    // the heads divide over the 8 XCDs, else the whole GPU).  Key steps per
    // query tile: the keys its last row sees (queued-causal), or the history
    // plus the queued chunks its rows span (isolated).
    const int wL = Tk - Tq;
    std::vector<int> steps(nqt);
    for (int qt = 0; qt < nqt; ++qt) {
      const int r0 = qt * ch.bm, r1 = std::min(Tq, r0 + ch.bm) - 1;
      const long long keys = isolated ? (long long)wL + (long long)(r1 / qlen + 1 - r0 / qlen) * qlen
                                      : (long long)wL + (long long)(r1 / qlen + 1) * qlen;
      steps[qt] = (int)((keys + ch.bk - 1) / ch.bk);
    }
    const double t_step = 4.0 * ch.bm * ch.bk * D / (flops / slots);  // one key step of one workgroup
    const double o_wg = 1.0;                                           // prologue and epilogue, in steps
    // a partial written at the CU's share of HBM bandwidth, in steps
    const double o_part = ch.bm * (D + 2) * 4.0 / (4.0e12 / cus) / t_step;
    const bool per_xcd = BH % 8 == 0;
    const int heads = per_xcd ? BH / 8 : BH;
    const int sl = (int)slots / (per_xcd ? 8 : 1);
    // more than four rounds of workgroups gain nothing; at most 48 whole-tile
    // counts per split count are priced (every one up to 48 query tiles)
    const int ns_cap = std::min(ns_max, std::max(8, (int)std::ceil(4.0 * slots / base)));
    const int stride = (nqt + 47) / 48;
    for (int ns = 1; ns <= ns_cap; ++ns) {
      for (int whole = ns == 1 ? nqt : 0; whole <= (ns == 1 ? nqt : nqt - 1); whole += (ns == 1 ? 1 : stride)) {
        const int rows = fwd_split_rows(ch.bm, Tq, SplitPlan{ns, whole});
        if (ns > 1 && fwd_split_bytes(D, BH, rows, ns) > ws_bytes) continue;
        const double t = split_makespan(steps, heads, sl, ns, whole, o_wg, o_part) * t_step +
                         (ns > 1 ? part_time(rows, ns) + 5e-6 : 0.0);  // merge traffic and its launch
        cands.push_back({t, {ns, ns > 1 ? whole : 0}});
      }
    }
  }
  // the simplest plan within 2% of the fastest: fewest splits, then most whole tiles
  double t_min = 1e300;
  for (const Cand& c : cands) t_min = std::min(t_min, c.t);
  SplitPlan best{1 << 30, 0};
  for (const Cand& c : cands) {
    if (c.t > t_min * 1.02) continue;
    if (c.sp.n_splits < best.n_splits || (c.sp.n_splits == best.n_splits && c.sp.n_whole > best.n_whole)) best = c.sp;
  }
  return best.n_splits == (1 << 30) ? SplitPlan{1, 0} : best;
}

}  // namespace

// Split plan from a cost model, memoised per shape (a streaming loop repeats
// its shape every step).  A call is bound by its MFMA time or by streaming
// its K/V window, whichever is larger at full occupancy.  A streaming-bound
// call splits every query tile and runs at the fraction of the 256 CUs its
// grid covers (one workgroup per CU keeps a CU's loads in flight).  For an
// MFMA-bound call a list-scheduling simulation of the dispatch order prices
// every split count and whole-tile count: keeping the heaviest tiles whole and
// splitting only the light ones that run last evens out the CUs' finish
// without the partials of a full split.  Each split adds fp32 partials, written
// and read back by the merge.  The plan taken is the simplest (fewest splits,
// then most whole tiles) within 2% of the fastest; each split keeps at least
// two key tiles; at most 64 splits; bounded by the workspace.  Measured
// on one queued chunk of 64-2640 tokens over a 6 x 2640 window it picks the
// fastest of 1-32 uniform splits.
SplitPlan fwd_plan_splits(const FwdChoice& ch, double flops, int kv_bytes, int D, int BH, int Tq, int Tk, int qlen,
                          bool isolated, size_t ws_bytes) {
  if (BH < 1 || Tq < 1 || Tk < 1 || qlen < 1 || ch.bm < 1 || ch.bk < 1) return {1, 0};
  static std::mutex mu;
  static std::map<PlanKey, SplitPlan> memo;
  const PlanKey key{ch.bm, ch.bk, ch.wg_per_cu, kv_bytes, D, BH, Tq, Tk, qlen, isolated ? 1 : 0, flops, ws_bytes};
  {
    std::lock_guard<std::mutex> lock(mu);
    auto it = memo.find(key);
    if (it != memo.end()) return it->second;
  }
  const SplitPlan sp = plan_splits(ch, flops, kv_bytes, D, BH, Tq, Tk, qlen, isolated, ws_bytes);
  std::lock_guard<std::mutex> lock(mu);
  if (memo.size() > 4096) memo.clear();
  memo[key] = sp;
  return sp;
}
#endif  // MW_FWD_HEAD_DIM == 128

}  // namespace mw
