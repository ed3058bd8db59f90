// Block-causal attention backward (gfx950): the analytic softmax gradient of
// paper Sec. 3.2's attention, with P recomputed from Q, K and the forward LSE.
//
//   row-term kernel : Delta_i = sum_d dO_id O_id                 (HBM-bound)
//   one grid of two kinds of workgroups:
//   dK/dV work : a workgroup owns 128 keys (32 per wave, K held in registers,
//                V in registers or, at D = 128, in an LDS tile); it walks the
//                query tiles that can see those keys -- queries of the same or
//                a later chunk -- staging Q, dO, LSE and Delta in LDS.  Per 32
//                queries and wave:
//                  S = Q K^T, dP = dO V^T     (keys on the lane axis)
//                  P = exp(S - LSE), dS = P (dP - Delta)
//                  dV^T += dO^T P, dK^T += Q^T dS   (transposing LDS reads)
//   dQ work    : a workgroup owns 128 queries (Q and dO in registers) and
//                walks the key tiles below the chunk diagonal:
//                  S^T = K Q^T, dP^T = V dO^T, dS^T = P^T (dP^T - Delta)
//                  dQ^T += K^T dS^T
// Recomputing S and dP in the dQ work costs 1.4x the MFMA work of a fused
// kernel with atomic dQ updates, but needs no fp32 dQ buffer and gives a
// deterministic result.
#include <type_traits>

#include "mw_device.h"
#include "mw_kernels.h"

namespace mw {

// Row terms of the backward pass: -Delta = -rowsum(dO * O) and LSE scaled to
// base 2 (LSE * log2 e), one 16-byte chunk per thread, reduced over the row's
// lanes.  Delta is stored negated: the dP products start from it (their MFMA
// accumulator input), so dP - Delta costs no instruction.
// CPR lanes per row (a power of two); at D = 72 the 9 pieces of a row leave
// lanes 9..15 of its group idle.
template <int D>
__global__ __launch_bounds__(256) void bwd_rowterms_kernel(BwdParams p, long long n_rows) {
  constexpr int CPR = D == 64 ? 8 : 16;
  const long long gid = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  const long long row = gid / CPR;
  const int c = (int)(gid % CPR);
  float acc = 0.f;
  if (row < n_rows && c < D / 8) {
    const long long bh = row / p.T, t = row - bh * p.T, bi = bh / p.H, hi = bh - bi * p.H;
    const u32x4 a = *reinterpret_cast<const u32x4*>(p.o + bi * p.so.b + hi * p.so.h + t * p.so.t + c * 8);
    const u32x4 b = *reinterpret_cast<const u32x4*>(p.d_o + bi * p.sdo.b + hi * p.sdo.h + t * p.sdo.t + c * 8);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const float a0 = __uint_as_float(a[j] << 16), a1 = __uint_as_float(a[j] & 0xffff0000u);
      const float b0 = __uint_as_float(b[j] << 16), b1 = __uint_as_float(b[j] & 0xffff0000u);
      acc = fmaf(a0, b0, acc);
      acc = fmaf(a1, b1, acc);
    }
  }
#pragma unroll
  for (int w = CPR / 2; w >= 1; w >>= 1) acc += __shfl_xor(acc, w);
  if (row < n_rows && c == 0) {
    p.delta[row] = -acc;
    p.lse2[row] = p.lse[row] * 1.4426950408889634f;
  }
}

// LDS of the dK/dV work: Q and dO tiles (two stages each), then LSE and -Delta
// of the tile's rows (two stages each, staged 64 rows at a time), then with
// VLDS the workgroup's V tile.
template <int D, int NW, int BM, int KBW, bool VLDS>
struct DkdvLds {
  static constexpr int TE = stage_elems<D, BM, 64 * NW>();
  static constexpr int RT = BM < 64 ? 64 : BM;  // row-term entries per stage
  static constexpr int TEV = VLDS ? stage_elems<D, 32 * NW * KBW, 64 * NW>() : 0;
  static constexpr int BYTES = 2 * 2 * TE * 2 + 2 * 2 * RT * 4 + TEV * 2;
};

// NW waves, each owning KBW blocks of 32 keys (K and V fragments and the dK,
// dV accumulators in registers).  With KBW = 2 every Q and dO fragment read
// from LDS feeds two MFMAs (one per key block), halving the LDS reads per
// MFMA; the register state then needs the full register file of one wave per
// SIMD (measured slower than one key block at two waves per SIMD at D = 64,
// where the in-order issue of a lone wave cannot overlap its MFMAs and its
// softmax work).  With VLDS the V fragments (the dP products' B operand) are
// read from the workgroup's V tile, staged in LDS once, instead of being held
// in registers: 32 registers fewer per wave at D = 128 for one more 1 KB
// fragment read per 32 x 32 block.  Work item: key tile kt of (batch, head) bh.
template <int D, int NW, int BM, int KBW, bool VLDS>
__device__ __forceinline__ void dkdv_body(const BwdParams& p, const int bh, const int kt, unsigned char* lds) {
  constexpr int BN = 32 * NW * KBW, NT = 64 * NW;
  static_assert(BM % 32 == 0, "32-row query blocks");
  static_assert(!VLDS || D % 16 == 0, "the V tile in LDS has no zero columns past D");
  constexpr int KK = (D + 15) / 16, DB = (D + 31) / 32;  // D = 72: 80 and 96 columns
  using LD = DkdvLds<D, NW, BM, KBW, VLDS>;
  constexpr int TE = LD::TE, RT = LD::RT;
  bf16_t(*Qs)[TE] = reinterpret_cast<bf16_t(*)[TE]>(lds);
  bf16_t(*dOs)[TE] = reinterpret_cast<bf16_t(*)[TE]>(lds + 2 * TE * 2);
  float(*lse_s)[RT] = reinterpret_cast<float(*)[RT]>(lds + 4 * TE * 2);
  float(*dlt_s)[RT] = reinterpret_cast<float(*)[RT]>(lds + 4 * TE * 2 + 2 * RT * 4);
  bf16_t* Vs = reinterpret_cast<bf16_t*>(lds + 4 * TE * 2 + 4 * RT * 4);  // (VLDS) the workgroup's V tile
  const FragOffsets<D> fo(threadIdx.x & 63, 0);  // Q and dO tiles share the layout

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int T = p.T, L = p.L;
  const int k0 = kt * BN;
  const int bi = bh / p.H, hi = bh - bi * p.H;
  const long long qb_ = bi * p.sq.b + hi * p.sq.h, dob_ = bi * p.sdo.b + hi * p.sdo.h;
  const float* lse2_bh = p.lse2 + (long long)bh * T;
  const float* dlt_bh = p.delta + (long long)bh * T;

  // Per key block: this lane's key, the first query that sees it, and its K and
  // V fragments (B operands of S = Q K^T and dP = dO V^T).  Keys past T read
  // the last key; their dK/dV are never stored.
  int mykey[KBW], qvis[KBW];
  bf16x8 kf[KBW][KK], vf[KBW][KK];
#pragma unroll
  for (int kb = 0; kb < KBW; ++kb) {
    mykey[kb] = k0 + (wave * KBW + kb) * 32 + (lane & 31);
    const long long kr = min(mykey[kb], T - 1);
    qvis[kb] = ((int)kr / L) * L;
    const bf16_t* ka = p.k + bi * p.sk.b + hi * p.sk.h + kr * p.sk.t + 8 * (lane >> 5);
    const bf16_t* va = p.v + bi * p.sv.b + hi * p.sv.h + kr * p.sv.t + 8 * (lane >> 5);
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
      if (D % 16 == 0 || 16 * kk + 8 * (lane >> 5) < D) {
        kf[kb][kk] = *reinterpret_cast<const bf16x8*>(ka + 16 * kk);
        if constexpr (!VLDS) vf[kb][kk] = *reinterpret_cast<const bf16x8*>(va + 16 * kk);
      } else {  // columns past D (D = 72): zeros
#pragma unroll
        for (int j = 0; j < 8; ++j) kf[kb][kk][j] = vf[kb][kk][j] = (__bf16)0.f;
      }
    }
  }
  f32x16 dv[KBW][DB], dk[KBW][DB];
#pragma unroll
  for (int kb = 0; kb < KBW; ++kb) {
#pragma unroll
    for (int db = 0; db < DB; ++db) {
      dv[kb][db] = zero16();
      dk[kb][db] = zero16();
    }
  }

  const int klast = min(k0 + BN, T) - 1;
  const int qstart = ((k0 / L) * L / BM) * BM;  // first query tile with a query of chunk >= chunk(k0)
  const float c = p.scale_log2;

  const RowOffsets<D, BM, NT> ro_q(p.sq.t, tid), ro_do(p.sdo.t, tid);
  auto stage = [&](int q0, int b) {
    if (q0 + BM <= T) {  // whole tile: scalar base + per-thread offsets
      stage_rows_s<D, BM, NT>(Qs[b], p.q + qb_ + q0 * p.sq.t, ro_q, tid);
      stage_rows_s<D, BM, NT>(dOs[b], p.d_o + dob_ + q0 * p.sdo.t, ro_do, tid);
    } else {  // the ragged last tile: rows past T read the last row
      stage_rows_direct<D, BM, NT>(Qs[b], [&](int r) { return p.q + qb_ + min(q0 + r, T - 1) * p.sq.t; }, tid);
      stage_rows_direct<D, BM, NT>(dOs[b], [&](int r) { return p.d_o + dob_ + min(q0 + r, T - 1) * p.sdo.t; }, tid);
    }
    // row terms of the tile: 64 fp32 per wave, LSE then -Delta
#pragma unroll
    for (int c = wave; c < 2 * (RT / 64); c += NW) {
      const int part = c % (RT / 64);
      if (c < RT / 64) {
        stage_f32x64_direct(lse_s[b] + 64 * part, lse2_bh, q0 + 64 * part, T, lane);
      } else {
        stage_f32x64_direct(dlt_s[b] + 64 * part, dlt_bh, q0 + 64 * part, T, lane);
      }
    }
  };

  auto step = [&](auto masked, const int q0, const int buf) {
    const bf16_t* Qt = Qs[buf];
    const bf16_t* dOt = dOs[buf];
#pragma unroll
    for (int qb = 0; qb < BM / 32; ++qb) {
      // -Delta of the tile's rows in accumulator layout (register i: row
      // 8(i/4) + 4(l/32) + i%4): the dP products accumulate onto it
      f32x16 ndl;
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const f32x4 d4 = *reinterpret_cast<const f32x4*>(&dlt_s[buf][qb * 32 + 8 * g + 4 * (lane >> 5)]);
#pragma unroll
        for (int j = 0; j < 4; ++j) ndl[4 * g + j] = d4[j];
      }
      f32x16 s[KBW], dp[KBW];
#pragma unroll
      for (int kb = 0; kb < KBW; ++kb) {
        s[kb] = zero16();
        dp[kb] = ndl;
      }
#pragma unroll
      for (int kk = 0; kk < KK; ++kk) {
        const bf16x8 qa = fo.row8(Qt, qb * 32, kk);
        const bf16x8 da = fo.row8(dOt, qb * 32, kk);
#pragma unroll
        for (int kb = 0; kb < KBW; ++kb) {
          s[kb] = mfma32(qa, kf[kb][kk], s[kb]);
          if constexpr (VLDS) {
            dp[kb] = mfma32(da, fo.row8(Vs, (wave * KBW + kb) * 32, kk), dp[kb]);
          } else {
            dp[kb] = mfma32(da, vf[kb][kk], dp[kb]);
          }
        }
      }
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int rr = qb * 32 + 8 * g + 4 * (lane >> 5);
        const f32x4 l4 = *reinterpret_cast<const f32x4*>(&lse_s[buf][rr]);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int i = 4 * g + j;
#pragma unroll
          for (int kb = 0; kb < KBW; ++kb) {
            float pv = fast_exp2(fmaf(s[kb][i], c, -l4[j]));
            if constexpr (decltype(masked)::value) {
              const int q = q0 + rr + j;
              const bool ok = (q < T) & (q >= qvis[kb]);  // q in the key's chunk or a later one
              pv = ok ? pv : 0.f;
            }
            s[kb][i] = pv;
            dp[kb][i] = pv * dp[kb][i];  // P (dP - Delta)
          }
        }
      }
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        bf16x8 pb[KBW], dsb[KBW];
#pragma unroll
        for (int kb = 0; kb < KBW; ++kb) {
          pb[kb] = pack8(s[kb], t);
          dsb[kb] = pack8(dp[kb], t);
        }
#pragma unroll
        for (int db = 0; db < DB; ++db) {
          const bf16x8 dot = fo.tr8(dOt, qb * 32, t, db);
#pragma unroll
          for (int kb = 0; kb < KBW; ++kb) dv[kb][db] = mfma32(dot, pb[kb], dv[kb][db]);
          const bf16x8 qt = fo.tr8(Qt, qb * 32, t, db);
#pragma unroll
          for (int kb = 0; kb < KBW; ++kb) dk[kb][db] = mfma32(qt, dsb[kb], dk[kb][db]);
        }
      }
    }
  };

  // Query tiles [qfb, qfe) see every key of this workgroup and are whole; the
  // ones before (same chunk as the keys) and the ragged last tile run masked.
  const int qfb = max(qstart, ((L * (klast / L) + BM - 1) / BM) * BM);
  const int qfe = max(qfb, (T / BM) * BM);
  int buf = 0;
  int q0 = qstart;
  if constexpr (VLDS) {  // the workgroup's V rows, read as the dP products' B operand
    const bf16_t* vb = p.v + bi * p.sv.b + hi * p.sv.h;
    if (k0 + BN <= T) {
      stage_rows_s<D, BN, NT>(Vs, vb + (long long)k0 * p.sv.t, RowOffsets<D, BN, NT>(p.sv.t, tid), tid);
    } else {
      stage_rows_direct<D, BN, NT>(Vs, [&](int r) { return vb + (long long)min(k0 + r, T - 1) * p.sv.t; }, tid);
    }
  }
  if (q0 < T) stage(q0, 0);
  wait_vmem();
  __syncthreads();
  auto run = [&](auto masked, const int qstop) {
    for (; q0 < qstop; q0 += BM) {
      if (q0 + BM < T) stage(q0 + BM, buf ^ 1);  // next query tile streams in during this one
      step(masked, q0, buf);
      wait_vmem();
      __syncthreads();
      buf ^= 1;
    }
  };
  run(std::true_type{}, min(qfb, T));
  run(std::false_type{}, min(qfe, T));
  run(std::true_type{}, T);

#pragma unroll
  for (int kb = 0; kb < KBW; ++kb) {
    if (mykey[kb] >= T) continue;
    bf16_t* dkrow = p.dk + bi * p.sdk.b + hi * p.sdk.h + mykey[kb] * p.sdk.t;
    bf16_t* dvrow = p.dv + bi * p.sdv.b + hi * p.sdv.h + mykey[kb] * p.sdv.t;
#pragma unroll
    for (int db = 0; db < DB; ++db) {
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        bf16x4 wk, wv;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          wk[j] = to_bf16(dk[kb][db][4 * g + j] * p.scale);
          wv[j] = to_bf16(dv[kb][db][4 * g + j]);
        }
        const int col = db * 32 + 8 * g + 4 * (lane >> 5);
        if (D % 32 != 0 && col >= D) continue;  // (D = 72)
        *reinterpret_cast<bf16x4*>(dkrow + col) = wk;
        *reinterpret_cast<bf16x4*>(dvrow + col) = wv;
      }
    }
  }
}

// LDS of the dQ work: K and V tiles, two stages each.
template <int D, int NW, int BN>
struct DqLds {
  static constexpr int TE = stage_elems<D, BN, 64 * NW>();
  static constexpr int BYTES = 2 * 2 * TE * 2;
};

// NW waves, each owning RB blocks of 32 query rows: with RB = 2 every K and V
// fragment read from LDS feeds two MFMAs (one per row block).  Work item:
// query tile qt of (batch, head) bh.
template <int D, int NW, int RB, int BN>
__device__ __forceinline__ void dq_body(const BwdParams& p, const int bh, const int qt, unsigned char* lds) {
  constexpr int BM = 32 * RB * NW, NT = 64 * NW;
  constexpr int KK = (D + 15) / 16, DB = (D + 31) / 32;  // D = 72: 80 and 96 columns
  constexpr int TE = DqLds<D, NW, BN>::TE;
  bf16_t(*Ks)[TE] = reinterpret_cast<bf16_t(*)[TE]>(lds);
  bf16_t(*Vs)[TE] = reinterpret_cast<bf16_t(*)[TE]>(lds + 2 * TE * 2);
  const FragOffsets<D> fo(threadIdx.x & 63, 0);  // K and V tiles share the layout

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int T = p.T, L = p.L;
  const int q0 = qt * BM;
  const int bi = bh / p.H, hi = bh - bi * p.H;
  const long long kb_ = bi * p.sk.b + hi * p.sk.h, vb_ = bi * p.sv.b + hi * p.sv.h;

  int qrow[RB], e1[RB];
  float lse2[RB], ndlt[RB];  // LSE * log2 e and -Delta of this lane's query
  bf16x8 qf[RB][KK], df[RB][KK];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    qrow[rb] = q0 + (wave * RB + rb) * 32 + (lane & 31);
    const int qc = min(qrow[rb], T - 1);
    const bf16_t* qa = p.q + bi * p.sq.b + hi * p.sq.h + qc * p.sq.t + 8 * (lane >> 5);
    const bf16_t* da = p.d_o + bi * p.sdo.b + hi * p.sdo.h + qc * p.sdo.t + 8 * (lane >> 5);
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
      if (D % 16 == 0 || 16 * kk + 8 * (lane >> 5) < D) {
        qf[rb][kk] = *reinterpret_cast<const bf16x8*>(qa + 16 * kk);
        df[rb][kk] = *reinterpret_cast<const bf16x8*>(da + 16 * kk);
      } else {  // columns past D (D = 72): zeros
#pragma unroll
        for (int j = 0; j < 8; ++j) qf[rb][kk][j] = df[rb][kk][j] = (__bf16)0.f;
      }
    }
    lse2[rb] = p.lse2[(long long)bh * T + qc];
    ndlt[rb] = p.delta[(long long)bh * T + qc];
    e1[rb] = min(T, (qc / L + 1) * L);
  }
  const int e1f = min(T, (q0 / L + 1) * L);
  const int kend = min(T, ((min(q0 + BM, T) - 1) / L + 1) * L);
  const float c = p.scale_log2;
  // -Delta depends only on the query (the lane's accumulator column): a tile
  // of it is the accumulator input of every dP product, so dS = P (dP - Delta)
  // is one multiply per element
  f32x16 ndl[RB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb)
#pragma unroll
    for (int i = 0; i < 16; ++i) ndl[rb][i] = ndlt[rb];

  f32x16 dq[RB][DB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb)
#pragma unroll
    for (int db = 0; db < DB; ++db) dq[rb][db] = zero16();

  const RowOffsets<D, BN, NT> ro_k(p.sk.t, tid), ro_v(p.sv.t, tid);
  auto stage = [&](int k0, int b) {
    if (k0 + BN <= T) {  // whole tile: scalar base + per-thread offsets
      stage_rows_s<D, BN, NT>(Ks[b], p.k + kb_ + k0 * p.sk.t, ro_k, tid);
      stage_rows_s<D, BN, NT>(Vs[b], p.v + vb_ + k0 * p.sv.t, ro_v, tid);
    } else {  // the ragged last tile: rows past T read the last row
      stage_rows_direct<D, BN, NT>(Ks[b], [&](int r) { return p.k + kb_ + min(k0 + r, T - 1) * p.sk.t; }, tid);
      stage_rows_direct<D, BN, NT>(Vs[b], [&](int r) { return p.v + vb_ + min(k0 + r, T - 1) * p.sv.t; }, tid);
    }
  };
  auto step = [&](auto masked, const int k0, const int buf) {
    const bf16_t* Kt = Ks[buf];
    const bf16_t* Vt = Vs[buf];
#pragma unroll
    for (int kb = 0; kb < BN / 32; ++kb) {
      f32x16 s[RB], dp[RB];
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) {
        s[rb] = zero16();
        dp[rb] = ndl[rb];
      }
#pragma unroll
      for (int kk = 0; kk < KK; ++kk) {
        const bf16x8 kfrag = fo.row8(Kt, kb * 32, kk);
        const bf16x8 vfrag = fo.row8(Vt, kb * 32, kk);
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) {
          s[rb] = mfma32(kfrag, qf[rb][kk], s[rb]);
          dp[rb] = mfma32(vfrag, df[rb][kk], dp[rb]);
        }
      }
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) {
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          float pv = fast_exp2(fmaf(s[rb][i], c, -lse2[rb]));
          if constexpr (decltype(masked)::value) {
            const int key = k0 + kb * 32 + acc_row(i, lane);
            pv = key < e1[rb] ? pv : 0.f;
          }
          dp[rb][i] = pv * dp[rb][i];  // P (dP - Delta)
        }
      }
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        bf16x8 dsb[RB];
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) dsb[rb] = pack8(dp[rb], t);
#pragma unroll
        for (int db = 0; db < DB; ++db) {
          const bf16x8 ktr = fo.tr8(Kt, kb * 32, t, db);
#pragma unroll
          for (int rb = 0; rb < RB; ++rb) dq[rb][db] = mfma32(ktr, dsb[rb], dq[rb][db]);
        }
      }
    }
  };

  // key tiles [0, kfull) are visible to every query of the workgroup
  const int kfull = (e1f / BN) * BN;
  int buf = 0;
  int k0 = 0;
  stage(0, 0);
  wait_vmem();
  __syncthreads();
  auto run = [&](auto masked, const int kstop) {
    for (; k0 < kstop; k0 += BN) {
      if (k0 + BN < kend) stage(k0 + BN, buf ^ 1);
      step(masked, k0, buf);
      wait_vmem();
      __syncthreads();
      buf ^= 1;
    }
  };
  run(std::false_type{}, min(kfull, kend));
  run(std::true_type{}, kend);

#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    if (qrow[rb] >= T) continue;
    bf16_t* row = p.dq + bi * p.sdq.b + hi * p.sdq.h + qrow[rb] * p.sdq.t;
#pragma unroll
    for (int db = 0; db < DB; ++db) {
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int col = db * 32 + 8 * g + 4 * (lane >> 5);
        if (D % 32 != 0 && col >= D) continue;  // (D = 72)
        bf16x4 w;
#pragma unroll
        for (int j = 0; j < 4; ++j) w[j] = to_bf16(dq[rb][db][4 * g + j] * p.scale);
        *reinterpret_cast<bf16x4*>(row + col) = w;
      }
    }
  }
}

// dK/dV and dQ work in one grid (both run two waves per SIMD with four-wave
// workgroups): the first n_dkdv workgroups take key tiles, the rest query
// tiles, so the query tiles fill the CUs that the key tiles' tail leaves idle
// and no kernel boundary separates them.  Each part keeps its own XCD-aware,
// heaviest-first order (tile_item; exact when n_dkdv is a multiple of the XCD
// count).  Early keys are seen by the most queries and late queries see the
// most keys: both parts run their heaviest tiles first.
template <int D, int NK, int BMK, int NQ, int RQ, int BNQ, bool VLDS>
__global__ __launch_bounds__(256, 2) void bwd_grad_kernel(BwdParams p, int n_dkdv, int n_ktiles, int n_qtiles) {
  static_assert(NK == 4 && NQ == 4, "four-wave workgroups");
  constexpr int B1 = DkdvLds<D, NK, BMK, 1, VLDS>::BYTES, B2 = DqLds<D, NQ, BNQ>::BYTES;
  __shared__ __attribute__((aligned(16))) unsigned char lds[B1 > B2 ? B1 : B2];
  const int id = blockIdx.x;
  int bh, r, split;
  if (id < n_dkdv) {
    tile_item(id, n_dkdv, p.BH, n_ktiles, 1, bh, r, split);
    dkdv_body<D, NK, BMK, 1, VLDS>(p, bh, r, lds);
  } else {
    tile_item(id - n_dkdv, (int)gridDim.x - n_dkdv, p.BH, n_qtiles, 1, bh, r, split);
    dq_body<D, NQ, RQ, BNQ>(p, bh, n_qtiles - 1 - r, lds);
  }
}

// Waves per workgroup of the dK/dV work (32 keys each) and of the dQ work (32
// queries each).
template <int D>
struct BwdCfg {
  static constexpr int NW_DKV = 4;
  static constexpr int NW_DQ = 4;
  // 32-row query blocks per wave in the dQ work (two measured no faster at
  // D = 64 and spill at D = 128)
  static constexpr int RB_DQ = 1;
  // D = 128: the V tile in LDS and 32-query steps bring the dK/dV work under
  // 256 registers (247), so it runs two waves per SIMD beside the dQ work in
  // one grid; holding V in registers needed 448 registers, one wave per SIMD,
  // in a grid of its own (the backward 5% slower, results bit-identical)
  static constexpr bool VLDS_DKV = D == 128;
  static constexpr int BM_DKV = D == 128 ? 32 : 64;  // queries per step of the dK/dV work
  static constexpr int BN_DQ = D == 64 ? 128 : 64;   // keys per step of the dQ work
};

template <int D>
static hipError_t launch_bwd_d(const BwdParams& p, hipStream_t stream) {
  constexpr int NK = BwdCfg<D>::NW_DKV, NQ = BwdCfg<D>::NW_DQ, RQ = BwdCfg<D>::RB_DQ;
  constexpr int BMK = BwdCfg<D>::BM_DKV, BNQ = BwdCfg<D>::BN_DQ;
  const long long rows = (long long)p.BH * p.T;
  const long long threads = rows * (D == 64 ? 8 : 16);
  hipLaunchKernelGGL(bwd_rowterms_kernel<D>, dim3((unsigned)((threads + 255) / 256)), dim3(256), 0, stream, p,
                     rows);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int nkt = (p.T + 32 * NK - 1) / (32 * NK);
  const int nqt = (p.T + 32 * RQ * NQ - 1) / (32 * RQ * NQ);
  hipLaunchKernelGGL((bwd_grad_kernel<D, NK, BMK, NQ, RQ, BNQ, BwdCfg<D>::VLDS_DKV>), dim3(nkt * p.BH + nqt * p.BH),
                     dim3(256), 0, stream, p, nkt * p.BH, nkt, nqt);
  return hipGetLastError();
}

// This file is compiled once per head dimension (MW_BWD_HEAD_DIM = 64, 72 or 128):
// the two instantiations get different instruction-scheduling options in the
// build (each measured the faster one for its size).
#if MW_BWD_HEAD_DIM == 64
hipError_t launch_bwd_64(const BwdParams& p, hipStream_t stream) { return launch_bwd_d<64>(p, stream); }
#elif MW_BWD_HEAD_DIM == 72
hipError_t launch_bwd_72(const BwdParams& p, hipStream_t stream) { return launch_bwd_d<72>(p, stream); }
#elif MW_BWD_HEAD_DIM == 128
hipError_t launch_bwd_128(const BwdParams& p, hipStream_t stream) { return launch_bwd_d<128>(p, stream); }
#else
#error "compile with -DMW_BWD_HEAD_DIM=64, 72 or 128"
#endif

}  // namespace mw
