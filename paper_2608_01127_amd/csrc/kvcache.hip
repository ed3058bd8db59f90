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
// `tab`.  One thread per (row, pair): a 4-byte load of the pair, an fp32
// rotation, a 4-byte store rounded to bf16.  HBM-bound.
__global__ __launch_bounds__(256) void rope_shift_kernel(uint16_t* __restrict__ k_slots, long long slot_stride, int S,
                                                         int first_slot, long long rows_per_slot, int D, int dim_offset,
                                                         int n_pairs, long long total, RopeTable tab) {
  const long long stride = (long long)gridDim.x * blockDim.x;
  for (long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += stride) {
    const int pair = (int)(i % n_pairs);
    const long long row = i / n_pairs;
    const long long ch = row / rows_per_slot, r = row % rows_per_slot;
    const int slot = (int)((first_slot + ch) % S);
    unsigned* w = reinterpret_cast<unsigned*>(k_slots + slot * slot_stride + r * D + dim_offset + 2 * pair);
    const unsigned u = *w;
    const float x0 = __uint_as_float(u << 16), x1 = __uint_as_float(u & 0xffff0000u);
    const float c = tab.c[pair], s = tab.s[pair];
    const float y0 = fmaf(x0, c, -x1 * s);
    const float y1 = fmaf(x0, s, x1 * c);
    const unsigned b0 = __builtin_bit_cast(unsigned short, to_bf16(y0));
    const unsigned b1 = __builtin_bit_cast(unsigned short, to_bf16(y1));
    *w = b0 | (b1 << 16);
  }
}

hipError_t launch_rope_shift(uint16_t* k_slots, long long slot_stride, int S, int first_slot, int n_live,
                             long long rows_per_slot, int D, int dim_offset, int n_pairs, const RopeTable& tab,
                             hipStream_t stream) {
  const long long total = (long long)n_live * rows_per_slot * n_pairs;
  long long blocks = (total + 255) / 256;
  if (blocks > 256 * 32) blocks = 256 * 32;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(rope_shift_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, k_slots, slot_stride, S,
                     first_slot, rows_per_slot, D, dim_offset, n_pairs, total, tab);
  return hipGetLastError();
}

hipError_t launch_kv_copy(const uint16_t* k_src, const uint16_t* v_src, uint16_t* k_dst, uint16_t* v_dst,
                          long long n_elems, hipStream_t stream) {
  const long long n16 = n_elems / 8;  // n_elems is a multiple of 8 (D is 64 or 128)
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
