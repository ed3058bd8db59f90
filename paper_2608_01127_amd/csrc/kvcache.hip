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

}  // namespace mw
