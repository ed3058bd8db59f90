// Commit copy of the rolling KV cache (paper Sec. 3.5): the keys and values of
// a chunk that reached the data endpoint are copied once into its ring slot
// and never modified afterwards.  Pure HBM traffic: 16-byte vector loads and
// stores, grid-stride, both tensors in one launch.
#include "mw_device.h"
#include "mw_kernels.h"

namespace mw {

__global__ __launch_bounds__(256) void kv_copy_kernel(const u32x4* __restrict__ ks, const u32x4* __restrict__ vs,
                                                      u32x4* __restrict__ kd, u32x4* __restrict__ vd, long long n16) {
  const long long stride = (long long)gridDim.x * blockDim.x;
  for (long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x; i < n16; i += stride) {
    const u32x4 a = __builtin_nontemporal_load(ks + i);
    const u32x4 b = __builtin_nontemporal_load(vs + i);
    kd[i] = a;
    vd[i] = b;
  }
}

// Commit of a strided chunk view: the destination slot is contiguous
// [B, H, L, D]; 16-byte pieces are gathered from the two source views.
__global__ __launch_bounds__(256) void kv_gather_kernel(const uint16_t* __restrict__ ks, const uint16_t* __restrict__ vs,
                                                        Strides sk, Strides sv, u32x4* __restrict__ kd,
                                                        u32x4* __restrict__ vd, int H, int L, int pieces_per_row,
                                                        long long n16) {
  const long long stride = (long long)gridDim.x * blockDim.x;
  for (long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x; i < n16; i += stride) {
    const long long row = i / pieces_per_row;
    const int c = (int)(i - row * pieces_per_row) * 8;
    const long long bh = row / L, t = row - bh * L, b = bh / H, h = bh - b * H;
    const u32x4 a = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(ks + b * sk.b + h * sk.h + t * sk.t + c));
    const u32x4 w = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(vs + b * sv.b + h * sv.h + t * sv.t + c));
    kd[i] = a;
    vd[i] = w;
  }
}

// RoPE re-shift of cached keys (paper Sec. 3.5): every key row of the live
// chunks gets its rope band rotated by the angles whose cos/sin the host put in
// `tab`.  Grid: (pieces of one slot / 256, live chunks), so the ring slot of a
// block is one scalar; one thread per 16-byte piece (4 pairs) of a row's band,
// read and written whole when the band starts on a 16-byte boundary, pair by
// pair otherwise and for a last piece of fewer than 4 pairs.  The cos/sin
// table is staged in LDS.  fp32 rotation, bf16 (RNE) stores.  HBM-bound.
__global__ __launch_bounds__(256) void rope_shift_kernel(uint16_t* __restrict__ k_slots, long long slot_stride, int S,
                                                         int first_slot, int rows_per_slot, int D, int dim_offset,
                                                         int n_pairs, RopeTable tab) {
  __shared__ float cs[2][64];
  if (threadIdx.x < 64) {
    cs[0][threadIdx.x] = tab.c[threadIdx.x];
    cs[1][threadIdx.x] = tab.s[threadIdx.x];
  }
  __syncthreads();
  const int ppr = (n_pairs + 3) >> 2;  // 16-byte pieces per row
  const int j = (int)blockIdx.x * 256 + (int)threadIdx.x;
  if (j >= rows_per_slot * ppr) return;
  const int slot = (first_slot + (int)blockIdx.y) % S;  // live chunk blockIdx.y, oldest first
  const int r = j / ppr, p0 = (j - r * ppr) * 4;
  uint16_t* w = k_slots + slot * slot_stride + (long long)r * D + dim_offset + 2 * p0;
  auto rot = [&](const unsigned u, const int pr) {
    const float x0 = __uint_as_float(u << 16), x1 = __uint_as_float(u & 0xffff0000u);
    const float c = cs[0][pr], sn = cs[1][pr];
    const float y0 = fmaf(x0, c, -x1 * sn);
    const float y1 = fmaf(x0, sn, x1 * c);
    const unsigned b0 = __builtin_bit_cast(unsigned short, to_bf16(y0));
    const unsigned b1 = __builtin_bit_cast(unsigned short, to_bf16(y1));
    return b0 | (b1 << 16);
  };
  if ((dim_offset & 7) == 0 && p0 + 4 <= n_pairs) {
    u32x4 v = *reinterpret_cast<const u32x4*>(w);
#pragma unroll
    for (int q = 0; q < 4; ++q) v[q] = rot(v[q], p0 + q);
    *reinterpret_cast<u32x4*>(w) = v;
  } else {
    unsigned* wp = reinterpret_cast<unsigned*>(w);
    for (int q = 0; q < 4 && p0 + q < n_pairs; ++q) wp[q] = rot(wp[q], p0 + q);
  }
}
hipError_t launch_rope_shift(uint16_t* k_slots, long long slot_stride, int S, int first_slot, int n_live,
                             long long rows_per_slot, int D, int dim_offset, int n_pairs, const RopeTable& tab,
                             hipStream_t stream) {
  const long long pieces = rows_per_slot * ((n_pairs + 3) / 4);
  if (n_live < 1 || pieces < 1) return hipSuccess;
  if (pieces > 0x7fffffffLL - 256 || n_live > 65535) return hipErrorInvalidValue;
  hipLaunchKernelGGL(rope_shift_kernel, dim3((unsigned)((pieces + 255) / 256), (unsigned)n_live), dim3(256), 0, stream,
                     k_slots, slot_stride, S, first_slot, (int)rows_per_slot, D, dim_offset, n_pairs, tab);
  return hipGetLastError();
}
hipError_t launch_kv_copy(const uint16_t* k_src, const uint16_t* v_src, uint16_t* k_dst, uint16_t* v_dst,
                          long long n_elems, hipStream_t stream) {
  const long long n16 = n_elems / 8;  // n_elems is a multiple of 8 (D is 64, 72 or 128)
  long long blocks = (n16 + 255) / 256;
  if (blocks > 256 * 16) blocks = 256 * 16;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(kv_copy_kernel, dim3((unsigned)blocks), dim3(256), 0, stream,
                     reinterpret_cast<const u32x4*>(k_src), reinterpret_cast<const u32x4*>(v_src),
                     reinterpret_cast<u32x4*>(k_dst), reinterpret_cast<u32x4*>(v_dst), n16);
  return hipGetLastError();
}

hipError_t launch_kv_gather(const uint16_t* k_src, const uint16_t* v_src, Strides sk, Strides sv, uint16_t* k_dst,
                            uint16_t* v_dst, int B, int H, int L, int D, hipStream_t stream) {
  const long long n16 = (long long)B * H * L * (D / 8);
  long long blocks = (n16 + 255) / 256;
  if (blocks > 256 * 16) blocks = 256 * 16;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(kv_gather_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, k_src, v_src, sk, sv,
                     reinterpret_cast<u32x4*>(k_dst), reinterpret_cast<u32x4*>(v_dst), H, L, D / 8, n16);
  return hipGetLastError();
}

}  // namespace mw
