// Block-causal attention backward (gfx950): the analytic softmax gradient of
// paper Sec. 3.2's attention, with P recomputed from Q, K and the forward LSE.
//
//   delta kernel : Delta_i = sum_d dO_id O_id                    (HBM-bound)
//   dK/dV kernel : one workgroup owns 128 keys (32 per wave, K and V held in
//                  registers); it walks the query tiles that can see those
//                  keys -- queries of the same or a later chunk -- staging Q,
//                  dO, LSE and Delta in LDS.  Per 32 queries and wave:
//                    S = Q K^T, dP = dO V^T     (keys on the lane axis)
//                    P = exp(S - LSE), dS = P (dP - Delta)
//                    dV^T += dO^T P, dK^T += Q^T dS   (transposing LDS reads)
//   dQ kernel    : one workgroup owns 128 queries (Q and dO in registers) and
//                  walks the key tiles below the chunk diagonal:
//                    S^T = K Q^T, dP^T = V dO^T, dS^T = P^T (dP^T - Delta)
//                    dQ^T += K^T dS^T
// Recomputing S and dP in the dQ kernel costs 1.4x the MFMA work of a fused
// kernel with atomic dQ updates, but needs no fp32 dQ buffer and gives a
// deterministic result.
#include "mw_device.h"
#include "mw_kernels.h"

namespace mw {

__device__ __forceinline__ int xcd_remap_b(int bid, int n) {
  if (n % 8) return bid;
  return (bid % 8) * (n / 8) + bid / 8;
}

// Delta = rowsum(dO * O): one 16-byte chunk per thread, reduced over the row's lanes.
template <int D>
__global__ __launch_bounds__(256) void bwd_delta_kernel(const uint16_t* __restrict__ o, const uint16_t* __restrict__ d_o,
                                                        float* __restrict__ delta, long long n_rows) {
  constexpr int CPR = D / 8;  // lanes per row (8 or 16)
  const long long gid = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  const long long row = gid / CPR;
  const int c = (int)(gid % CPR);
  float acc = 0.f;
  if (row < n_rows) {
    const u32x4 a = *reinterpret_cast<const u32x4*>(o + row * D + c * 8);
    const u32x4 b = *reinterpret_cast<const u32x4*>(d_o + row * D + c * 8);
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
  if (row < n_rows && c == 0) delta[row] = acc;
}

template <int D>
__global__ __launch_bounds__(256, 1) void bwd_dkdv_kernel(BwdParams p, int n_ktiles) {
  constexpr int BN = DKV_BN, BM = DKV_BM, NT = 256;
  constexpr int KK = D / 16, DB = D / 32, CPR = D / 8;
  __shared__ __attribute__((aligned(16))) bf16_t Qs[BM * D];
  __shared__ __attribute__((aligned(16))) bf16_t dOs[BM * D];
  __shared__ __attribute__((aligned(16))) float lse_s[BM];
  __shared__ __attribute__((aligned(16))) float dlt_s[BM];

  const int logical = xcd_remap_b(blockIdx.x, gridDim.x);
  const int bh = logical / n_ktiles;
  const int kt = logical % n_ktiles;  // early keys are seen by the most queries: heaviest first
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int T = p.T, L = p.L;
  const int k0 = kt * BN;
  const int mykey = k0 + wave * 32 + (lane & 31);
  const long long off = (long long)bh * T * D;

  // K and V fragments: B operands of S = Q K^T and dP = dO V^T.
  bf16x8 kf[KK], vf[KK];
#pragma unroll
  for (int kk = 0; kk < KK; ++kk) {
    if (mykey < T) {
      const long long a = off + (long long)mykey * D + 16 * kk + 8 * (lane >> 5);
      kf[kk] = *reinterpret_cast<const bf16x8*>(p.k + a);
      vf[kk] = *reinterpret_cast<const bf16x8*>(p.v + a);
    } else {
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        kf[kk][j] = (__bf16)0.f;
        vf[kk][j] = (__bf16)0.f;
      }
    }
  }
  f32x16 dv[DB], dk[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) {
    dv[db] = zero16();
    dk[db] = zero16();
  }

  const int klast = min(k0 + BN, T) - 1;
  const int qstart = ((k0 / L) * L / BM) * BM;  // first query tile with a query of chunk >= chunk(k0)
  const float c = p.scale_log2;

  for (int q0 = qstart; q0 < T; q0 += BM) {
    const bool full = (q0 / L) >= (klast / L);
    __syncthreads();
#pragma unroll
    for (int it = 0; it < BM * CPR / NT; ++it) {
      const int ci = tid + NT * it;
      const int r = ci / CPR, cc = (ci % CPR) * 8;
      const int q = q0 + r;
      u32x4 qv = {0, 0, 0, 0}, dov = {0, 0, 0, 0};
      if (q < T) {
        const long long a = off + (long long)q * D + cc;
        qv = *reinterpret_cast<const u32x4*>(p.q + a);
        dov = *reinterpret_cast<const u32x4*>(p.d_o + a);
      }
      *reinterpret_cast<u32x4*>(Qs + Tile<D>::off(r, cc)) = qv;
      *reinterpret_cast<u32x4*>(dOs + Tile<D>::off(r, cc)) = dov;
    }
    if (tid < BM) {
      const int q = q0 + tid;
      // padding rows get LSE = +inf, so their probabilities are exactly 0
      lse_s[tid] = q < T ? p.lse[(long long)bh * T + q] * 1.4426950408889634f : INFINITY;
      dlt_s[tid] = q < T ? p.delta[(long long)bh * T + q] : 0.f;
    }
    __syncthreads();

#pragma unroll
    for (int qb = 0; qb < BM / 32; ++qb) {
      f32x16 s = zero16(), dp = zero16();
#pragma unroll
      for (int kk = 0; kk < KK; ++kk) {
        s = mfma32(lds_row8<D>(Qs, qb * 32 + (lane & 31), 16 * kk + 8 * (lane >> 5)), kf[kk], s);
        dp = mfma32(lds_row8<D>(dOs, qb * 32 + (lane & 31), 16 * kk + 8 * (lane >> 5)), vf[kk], dp);
      }
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int rr = qb * 32 + 8 * g + 4 * (lane >> 5);
        const f32x4 l4 = *reinterpret_cast<const f32x4*>(lse_s + rr);
        const f32x4 d4 = *reinterpret_cast<const f32x4*>(dlt_s + rr);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          const int i = 4 * g + j;
          float pv = exp2f(fmaf(s[i], c, -l4[j]));
          if (!full) {
            const int q = q0 + rr + j;
            const int e1 = min(T, (q / L + 1) * L);
            pv = mykey < e1 ? pv : 0.f;
          }
          s[i] = pv;
          dp[i] = pv * (dp[i] - d4[j]);
        }
      }
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        const bf16x8 pb = pack8(s, t);
        const bf16x8 dsb = pack8(dp, t);
#pragma unroll
        for (int db = 0; db < DB; ++db) {
          dv[db] = mfma32(lds_tr8<D>(dOs, qb * 32, t, db * 32, lane), pb, dv[db]);
          dk[db] = mfma32(lds_tr8<D>(Qs, qb * 32, t, db * 32, lane), dsb, dk[db]);
        }
      }
    }
  }

  if (mykey < T) {
    bf16_t* dkrow = p.dk + off + (long long)mykey * D;
    bf16_t* dvrow = p.dv + off + (long long)mykey * D;
#pragma unroll
    for (int db = 0; db < DB; ++db) {
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        bf16x4 wk, wv;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          wk[j] = to_bf16(dk[db][4 * g + j] * p.scale);
          wv[j] = to_bf16(dv[db][4 * g + j]);
        }
        const int col = db * 32 + 8 * g + 4 * (lane >> 5);
        *reinterpret_cast<bf16x4*>(dkrow + col) = wk;
        *reinterpret_cast<bf16x4*>(dvrow + col) = wv;
      }
    }
  }
}

template <int D>
__global__ __launch_bounds__(256, 2) void bwd_dq_kernel(BwdParams p, int n_qtiles) {
  constexpr int BM = DQ_BM, BN = DQ_BN, NT = 256;
  constexpr int KK = D / 16, DB = D / 32, CPR = D / 8;
  __shared__ __attribute__((aligned(16))) bf16_t Ks[BN * D];
  __shared__ __attribute__((aligned(16))) bf16_t Vs[BN * D];

  const int logical = xcd_remap_b(blockIdx.x, gridDim.x);
  const int bh = logical / n_qtiles;
  const int qt = n_qtiles - 1 - logical % n_qtiles;  // late queries see the most keys: heaviest first
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int T = p.T, L = p.L;
  const int q0 = qt * BM;
  const int qrow = q0 + wave * 32 + (lane & 31);
  const long long off = (long long)bh * T * D;

  bf16x8 qf[KK], df[KK];
#pragma unroll
  for (int kk = 0; kk < KK; ++kk) {
    if (qrow < T) {
      const long long a = off + (long long)qrow * D + 16 * kk + 8 * (lane >> 5);
      qf[kk] = *reinterpret_cast<const bf16x8*>(p.q + a);
      df[kk] = *reinterpret_cast<const bf16x8*>(p.d_o + a);
    } else {
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        qf[kk][j] = (__bf16)0.f;
        df[kk][j] = (__bf16)0.f;
      }
    }
  }
  const float lse2 = qrow < T ? p.lse[(long long)bh * T + qrow] * 1.4426950408889634f : INFINITY;
  const float dlt = qrow < T ? p.delta[(long long)bh * T + qrow] : 0.f;
  const int e1 = min(T, (min(qrow, T - 1) / L + 1) * L);
  const int e1f = min(T, (q0 / L + 1) * L);
  const int kend = min(T, ((min(q0 + BM, T) - 1) / L + 1) * L);
  const float c = p.scale_log2;

  f32x16 dq[DB];
#pragma unroll
  for (int db = 0; db < DB; ++db) dq[db] = zero16();

  for (int k0 = 0; k0 < kend; k0 += BN) {
    const bool full = k0 + BN <= e1f;
    __syncthreads();
#pragma unroll
    for (int it = 0; it < BN * CPR / NT; ++it) {
      const int ci = tid + NT * it;
      const int r = ci / CPR, cc = (ci % CPR) * 8;
      const int key = k0 + r;
      u32x4 kv = {0, 0, 0, 0}, vv = {0, 0, 0, 0};
      if (key < T) {
        const long long a = off + (long long)key * D + cc;
        kv = *reinterpret_cast<const u32x4*>(p.k + a);
        vv = *reinterpret_cast<const u32x4*>(p.v + a);
      }
      *reinterpret_cast<u32x4*>(Ks + Tile<D>::off(r, cc)) = kv;
      *reinterpret_cast<u32x4*>(Vs + Tile<D>::off(r, cc)) = vv;
    }
    __syncthreads();

#pragma unroll
    for (int kb = 0; kb < BN / 32; ++kb) {
      f32x16 s = zero16(), dp = zero16();
#pragma unroll
      for (int kk = 0; kk < KK; ++kk) {
        s = mfma32(lds_row8<D>(Ks, kb * 32 + (lane & 31), 16 * kk + 8 * (lane >> 5)), qf[kk], s);
        dp = mfma32(lds_row8<D>(Vs, kb * 32 + (lane & 31), 16 * kk + 8 * (lane >> 5)), df[kk], dp);
      }
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        float pv = exp2f(fmaf(s[i], c, -lse2));
        if (!full) {
          const int key = k0 + kb * 32 + acc_row(i, lane);
          pv = key < e1 ? pv : 0.f;
        }
        dp[i] = pv * (dp[i] - dlt);
      }
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        const bf16x8 dsb = pack8(dp, t);
#pragma unroll
        for (int db = 0; db < DB; ++db) dq[db] = mfma32(lds_tr8<D>(Ks, kb * 32, t, db * 32, lane), dsb, dq[db]);
      }
    }
  }

  if (qrow < T) {
    bf16_t* row = p.dq + off + (long long)qrow * D;
#pragma unroll
    for (int db = 0; db < DB; ++db) {
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        bf16x4 w;
#pragma unroll
        for (int j = 0; j < 4; ++j) w[j] = to_bf16(dq[db][4 * g + j] * p.scale);
        *reinterpret_cast<bf16x4*>(row + db * 32 + 8 * g + 4 * (lane >> 5)) = w;
      }
    }
  }
}

template <int D>
static hipError_t launch_bwd_d(const BwdParams& p, hipStream_t stream) {
  const long long rows = (long long)p.BH * p.T;
  const long long threads = rows * (D / 8);
  hipLaunchKernelGGL(bwd_delta_kernel<D>, dim3((unsigned)((threads + 255) / 256)), dim3(256), 0, stream, p.o, p.d_o,
                     p.delta, rows);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int nkt = (p.T + DKV_BN - 1) / DKV_BN;
  hipLaunchKernelGGL(bwd_dkdv_kernel<D>, dim3(nkt * p.BH), dim3(256), 0, stream, p, nkt);
  e = hipGetLastError();
  if (e != hipSuccess) return e;
  const int nqt = (p.T + DQ_BM - 1) / DQ_BM;
  hipLaunchKernelGGL(bwd_dq_kernel<D>, dim3(nqt * p.BH), dim3(256), 0, stream, p, nqt);
  return hipGetLastError();
}

hipError_t launch_bwd(const BwdParams& p, int D, hipStream_t stream) {
  return D == 64 ? launch_bwd_d<64>(p, stream) : launch_bwd_d<128>(p, stream);
}

}  // namespace mw
