// C ABI of the library (declared in include/mw.h): argument validation, ring
// bookkeeping and kernel launches.  No device memory is allocated here.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdint>
#include <cstdio>
#include <mutex>
#include <string>

#include "mw.h"
#include "mw_kernels.h"

namespace {

thread_local std::string g_err;

int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

int ok() {
  g_err.clear();
  return MW_OK;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

constexpr int kMaxT = 1 << 24;  // keeps every in-kernel row * D index within 32 bits

int check_ptrs(const char* fn, std::initializer_list<std::pair<const char*, const void*>> ptrs) {
  for (auto& pr : ptrs)
    if (pr.second == nullptr) return fail(MW_EINVAL, "%s: %s is NULL", fn, pr.first);
  for (auto& pr : ptrs)
    if (!aligned16(pr.second)) return fail(MW_EALIGN, "%s: %s is not 16-byte aligned", fn, pr.first);
  return MW_OK;
}

int check_train_dims(const char* fn, int B, int H, int T, int D, int chunk_len, float scale) {
  if (B < 1 || H < 1 || T < 1 || chunk_len < 1)
    return fail(MW_EINVAL, "%s: B, H, T and chunk_len must be >= 1 (got %d, %d, %d, %d)", fn, B, H, T, chunk_len);
  if (D != 64 && D != 72 && D != 128)
    return fail(MW_EUNSUPPORTED, "%s: head dimension %d is not supported (64, 72 or 128)", fn, D);
  if (T > kMaxT) return fail(MW_EUNSUPPORTED, "%s: T = %d exceeds %d", fn, T, kMaxT);
  if ((long long)B * H > (1LL << 24)) return fail(MW_EUNSUPPORTED, "%s: B*H too large", fn);
  if (!(scale > 0.f) || !std::isfinite(scale)) return fail(MW_EINVAL, "%s: scale must be finite and > 0", fn);
  return MW_OK;
}

int hip_status(const char* fn, hipError_t e) {
  if (e != hipSuccess) return fail(MW_EHIP, "%s: HIP error %s", fn, hipGetErrorString(e));
  return ok();
}

const float kLog2e = 1.4426950408889634f;

mw::Strides contiguous(int H, int T, int D) { return {(long long)H * T * D, (long long)T * D, D}; }

// A [B, H, T, D] view with D contiguous: strides non-negative, rows 16-byte
// aligned (every stride a multiple of 8 elements), rows at least D apart.
// Output views must also not overlap themselves: sorted by stride, each
// dimension must step past everything the smaller ones span.
int check_view(const char* fn, const char* name, const mw_strides& s, int B, int H, int T, int D, bool output) {
  if (s.b < 0 || s.h < 0 || s.t < D)
    return fail(MW_EINVAL, "%s: strides of %s must be >= 0 with a T stride >= D (got %lld, %lld, %lld)", fn, name,
                (long long)s.b, (long long)s.h, (long long)s.t);
  if (s.b % 8 || s.h % 8 || s.t % 8)
    return fail(MW_EALIGN, "%s: strides of %s must be multiples of 8 elements (16-byte rows)", fn, name);
  if (s.t > (1LL << 23))  // byte offsets within a staged tile of up to 128 rows stay below 2^32
    return fail(MW_EUNSUPPORTED, "%s: T stride of %s exceeds 2^23 elements", fn, name);
  const long double span = (long double)(B - 1) * s.b + (long double)(H - 1) * s.h + (long double)(T - 1) * s.t + D;
  if (span > (long double)(1LL << 60)) return fail(MW_EUNSUPPORTED, "%s: view %s spans too many elements", fn, name);
  if (!output) return MW_OK;
  struct Dim {
    long long stride, extent;
  } dims[3] = {{s.t, T}, {s.h, H}, {s.b, B}};
  for (int i = 0; i < 3; ++i)  // sort by stride (three elements)
    for (int j = i + 1; j < 3; ++j)
      if (dims[j].stride < dims[i].stride) {
        Dim t = dims[i];
        dims[i] = dims[j];
        dims[j] = t;
      }
  long long covered = D;  // elements spanned by the dimensions below
  for (auto& d : dims) {
    if (d.extent == 1) continue;
    if (d.stride < covered) return fail(MW_EINVAL, "%s: output view %s overlaps itself", fn, name);
    covered = d.stride * (d.extent - 1) + covered;
  }
  return MW_OK;
}

mw::Strides to_internal(const mw_strides& s) { return {s.b, s.h, s.t}; }

}  // namespace

namespace mw {
int set_error(int code, const char* msg) {
  g_err = code == MW_OK ? std::string() : std::string(msg);
  return code;
}
}  // namespace mw

extern "C" {

const char* mw_last_error(void) { return g_err.c_str(); }

int mw_version(void) { return 100; }

int mw_block_causal_attn_fwd_strided(const void* q, const void* k, const void* v, void* o, float* lse,
                                     const mw_strides* strides, int B, int H, int T, int D, int chunk_len,
                                     float scale, mw_stream_t stream) {
  const char* fn = "mw_block_causal_attn_fwd";
  int st = check_ptrs(fn, {{"q", q}, {"k", k}, {"v", v}, {"o", o}, {"lse", lse}});
  if (st) return st;
  st = check_train_dims(fn, B, H, T, D, chunk_len, scale);
  if (st) return st;
  mw::Strides sv[4];
  const char* names[4] = {"q", "k", "v", "o"};
  for (int i = 0; i < 4; ++i) {
    if (strides == nullptr) {
      sv[i] = contiguous(H, T, D);
      continue;
    }
    st = check_view(fn, names[i], strides[i], B, H, T, D, i == 3);
    if (st) return st;
    sv[i] = to_internal(strides[i]);
  }
  mw::FwdParams p{};
  p.q = static_cast<const uint16_t*>(q);
  p.k = static_cast<const uint16_t*>(k);
  p.v = static_cast<const uint16_t*>(v);
  p.o = static_cast<uint16_t*>(o);
  p.lse = lse;
  p.BH = B * H;
  p.H = H;
  p.Tq = T;
  p.vis_mode = 0;
  p.L = chunk_len > T ? T : chunk_len;
  p.Tk = T;
  p.qlen = 1;
  p.wL = 0;
  p.scale_log2 = scale * kLog2e;
  p.scale_ln = scale;
  p.sq = sv[0];
  p.sk = sv[1];
  p.sv = sv[2];
  p.so = sv[3];
  return hip_status(fn, mw::launch_fwd(p, D, false, static_cast<hipStream_t>(stream)));
}

int mw_block_causal_attn_fwd(const void* q, const void* k, const void* v, void* o, float* lse, int B, int H, int T,
                             int D, int chunk_len, float scale, mw_stream_t stream) {
  return mw_block_causal_attn_fwd_strided(q, k, v, o, lse, nullptr, B, H, T, D, chunk_len, scale, stream);
}

size_t mw_block_causal_attn_bwd_workspace_size(int B, int H, int T, int D) {
  (void)D;
  if (B < 1 || H < 1 || T < 1) return 0;
  const size_t bytes = (size_t)B * H * T * sizeof(float);
  return 2 * ((bytes + 255) & ~(size_t)255);  // -Delta and base-2 LSE, one fp32 per row each
}

int mw_block_causal_attn_bwd_strided(const void* q, const void* k, const void* v, const void* o, const void* d_o,
                                     const float* lse, void* dq, void* dk, void* dv, void* workspace,
                                     size_t workspace_bytes, const mw_strides* strides, int B, int H, int T, int D,
                                     int chunk_len, float scale, mw_stream_t stream) {
  const char* fn = "mw_block_causal_attn_bwd";
  int st = check_ptrs(fn, {{"q", q}, {"k", k}, {"v", v}, {"o", o}, {"d_o", d_o}, {"lse", lse}, {"dq", dq},
                           {"dk", dk}, {"dv", dv}, {"workspace", workspace}});
  if (st) return st;
  st = check_train_dims(fn, B, H, T, D, chunk_len, scale);
  if (st) return st;
  const size_t need = mw_block_causal_attn_bwd_workspace_size(B, H, T, D);
  if (workspace_bytes < need)
    return fail(MW_EINVAL, "%s: workspace of %zu bytes is smaller than the %zu bytes needed", fn, workspace_bytes,
                need);
  mw::Strides sv[8];
  const char* names[8] = {"q", "k", "v", "o", "d_o", "dq", "dk", "dv"};
  for (int i = 0; i < 8; ++i) {
    if (strides == nullptr) {
      sv[i] = contiguous(H, T, D);
      continue;
    }
    st = check_view(fn, names[i], strides[i], B, H, T, D, i >= 5);
    if (st) return st;
    sv[i] = to_internal(strides[i]);
  }
  mw::BwdParams p{};
  p.q = static_cast<const uint16_t*>(q);
  p.k = static_cast<const uint16_t*>(k);
  p.v = static_cast<const uint16_t*>(v);
  p.o = static_cast<const uint16_t*>(o);
  p.d_o = static_cast<const uint16_t*>(d_o);
  p.lse = lse;
  p.delta = static_cast<float*>(workspace);
  p.lse2 = reinterpret_cast<float*>(static_cast<char*>(workspace) + need / 2);
  p.dq = static_cast<uint16_t*>(dq);
  p.dk = static_cast<uint16_t*>(dk);
  p.dv = static_cast<uint16_t*>(dv);
  p.BH = B * H;
  p.H = H;
  p.T = T;
  p.L = chunk_len > T ? T : chunk_len;
  p.scale = scale;
  p.scale_log2 = scale * kLog2e;
  p.sq = sv[0];
  p.sk = sv[1];
  p.sv = sv[2];
  p.so = sv[3];
  p.sdo = sv[4];
  p.sdq = sv[5];
  p.sdk = sv[6];
  p.sdv = sv[7];
  hipStream_t hs = static_cast<hipStream_t>(stream);
  return hip_status(fn, D == 64 ? mw::launch_bwd_64(p, hs) : (D == 72 ? mw::launch_bwd_72(p, hs) : mw::launch_bwd_128(p, hs)));
}

int mw_block_causal_attn_bwd(const void* q, const void* k, const void* v, const void* o, const void* d_o,
                             const float* lse, void* dq, void* dk, void* dv, void* workspace, size_t workspace_bytes,
                             int B, int H, int T, int D, int chunk_len, float scale, mw_stream_t stream) {
  return mw_block_causal_attn_bwd_strided(q, k, v, o, d_o, lse, dq, dk, dv, workspace, workspace_bytes, nullptr, B, H,
                                          T, D, chunk_len, scale, stream);
}

// ---------------------------------------------------------------------------
// The backward without a caller workspace.  Its row terms (-Delta and the
// base-2 LSE, 8 bytes per row) live in `scratch`, a fixed device array of this
// library: every GPU the library runs on holds one copy of it for the life of
// the process.  In host code the array's name stands for a host-side shadow,
// so the device copy's address is asked of the runtime once per device and
// only that address is ever handed to kernels.
// ---------------------------------------------------------------------------
namespace {

constexpr size_t kScratchBytes = size_t(32) << 20;  // 2 x 16 MiB: up to 4,194,304 rows (B * H * T)
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// Device address of the current device's copy of `scratch` (looked up on the
// first call on that device, with the device current).
int scratch_address(const char* fn, void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(MW_EHIP, "%s: hipGetDevice failed: %s", fn, hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices) return fail(MW_EUNSUPPORTED, "%s: device %d is beyond %d", fn, dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_ptr[dev] == nullptr) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || p == nullptr)
      return fail(MW_EHIP, "%s: no device address for the scratch array on device %d: %s", fn, dev,
                  hipGetErrorString(e));
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return MW_OK;
}

}  // namespace

int mw_block_causal_attn_bwd_noalloc(const void* q, const void* k, const void* v, const void* o, const void* d_o,
                                     const float* lse, void* dq, void* dk, void* dv, int B, int H, int T, int D,
                                     int chunk_len, float scale, mw_stream_t stream) {
  const char* fn = "mw_block_causal_attn_bwd_noalloc";
  int st = check_ptrs(fn, {{"q", q}, {"k", k}, {"v", v}, {"o", o}, {"d_o", d_o}, {"lse", lse}, {"dq", dq},
                           {"dk", dk}, {"dv", dv}});
  if (st) return st;
  st = check_train_dims(fn, B, H, T, D, chunk_len, scale);
  if (st) return st;
  const size_t need = mw_block_causal_attn_bwd_workspace_size(B, H, T, D);
  if (need > kScratchBytes)
    return fail(MW_EUNSUPPORTED, "%s: B*H*T = %lld rows need %zu bytes of row terms, beyond the library's %zu-byte "
                "scratch array (at most %zu rows)", fn, (long long)B * H * T, need, kScratchBytes,
                kScratchBytes / (2 * sizeof(float)));
  void* ws = nullptr;
  st = scratch_address(fn, &ws);
  if (st) return st;
  return mw_block_causal_attn_bwd_strided(q, k, v, o, d_o, lse, dq, dk, dv, ws, kScratchBytes, nullptr, B, H, T, D,
                                          chunk_len, scale, stream);
}

int mw_kvcache_init(mw_kvcache* c, void* k_slots, void* v_slots, int S, int B, int H, int L, int D) {
  const char* fn = "mw_kvcache_init";
  if (c == nullptr) return fail(MW_EINVAL, "%s: cache is NULL", fn);
  int st = check_ptrs(fn, {{"k_slots", k_slots}, {"v_slots", v_slots}});
  if (st) return st;
  if (S < 1 || B < 1 || H < 1 || L < 1)
    return fail(MW_EINVAL, "%s: S, B, H and L must be >= 1 (got %d, %d, %d, %d)", fn, S, B, H, L);
  if (D != 64 && D != 72 && D != 128)
    return fail(MW_EUNSUPPORTED, "%s: head dimension %d is not supported (64, 72 or 128)", fn, D);
  if ((long long)L * S > kMaxT) return fail(MW_EUNSUPPORTED, "%s: S*L exceeds %d tokens", fn, kMaxT);
  c->k_slots = k_slots;
  c->v_slots = v_slots;
  c->S = S;
  c->B = B;
  c->H = H;
  c->L = L;
  c->D = D;
  c->head = 0;
  c->tail = 0;
  c->k_sink = nullptr;
  c->v_sink = nullptr;
  c->sink_len = 0;
  c->elem_bytes = 2;
  c->k_scale = 1.f;
  c->v_scale = 1.f;
  c->rope_total = 0;
  c->rope_offset = 0;
  c->rope_count = 0;
  c->rope_theta = 0.f;
  c->rope_set = 0;
  for (int i = 0; i < MW_MAX_SLOTS; ++i) c->rope_at_commit[i] = 0;
  return ok();
}

static bool good_scale(float s) { return s > 0.f && std::isfinite(s); }

int mw_kvcache_init_fp8(mw_kvcache* c, void* k_slots, void* v_slots, int S, int B, int H, int L, int D, float k_scale,
                        float v_scale) {
  const char* fn = "mw_kvcache_init_fp8";
  if (c == nullptr) return fail(MW_EINVAL, "%s: cache is NULL", fn);
  if (D != 128) return fail(MW_EUNSUPPORTED, "%s: head dimension %d is not supported (128)", fn, D);
  if (!good_scale(k_scale) || !good_scale(v_scale))
    return fail(MW_EINVAL, "%s: k_scale and v_scale must be finite and > 0", fn);
  if (S > MW_MAX_SLOTS) return fail(MW_EUNSUPPORTED, "%s: S = %d exceeds %d slots", fn, S, MW_MAX_SLOTS);
  mw_kvcache t;
  const int st = mw_kvcache_init(&t, k_slots, v_slots, S, B, H, L, D);
  if (st) return fail(st, "%s: %s", fn, mw_last_error());
  t.elem_bytes = 1;
  t.k_scale = k_scale;
  t.v_scale = v_scale;
  *c = t;
  return ok();
}

static int check_cache(const char* fn, const mw_kvcache* c) {
  if (c == nullptr) return fail(MW_EINVAL, "%s: cache is NULL", fn);
  if (c->k_slots == nullptr || c->v_slots == nullptr || c->S < 1 || c->B < 1 || c->H < 1 || c->L < 1 ||
      (c->D != 64 && c->D != 72 && c->D != 128) || c->tail < 0 || c->head < c->tail || c->head - c->tail > c->S ||
      c->sink_len < 0 || (c->sink_len > 0 && (c->k_sink == nullptr || c->v_sink == nullptr)) ||
      (c->elem_bytes != 1 && c->elem_bytes != 2) ||
      (c->elem_bytes == 1 && (c->D != 128 || !good_scale(c->k_scale) || !good_scale(c->v_scale) ||
                              c->S > MW_MAX_SLOTS)) ||
      (c->rope_set != 0 && c->rope_set != 1))
    return fail(MW_EINVAL, "%s: cache descriptor is not initialised or is corrupt", fn);
  return MW_OK;
}

// A RoPE band of `D` head dims: even offset, even count of 2..128 dims, inside D.
static int check_band(const char* fn, const mw_rope* rope, int D) {
  if (rope->dim_offset < 0 || rope->dim_offset % 2 || rope->dim_count < 2 || rope->dim_count % 2 ||
      rope->dim_count > 128 || rope->dim_offset + rope->dim_count > D)
    return fail(MW_EINVAL, "%s: rope band [%d, %d) is not a valid even band of the %d head dims", fn, rope->dim_offset,
                rope->dim_offset + rope->dim_count, D);
  if (!(rope->theta > 0.f) || !std::isfinite(rope->theta)) return fail(MW_EINVAL, "%s: theta must be > 0", fn);
  return MW_OK;
}

int mw_kvcache_append_strided(mw_kvcache* c, const void* k_chunk, const void* v_chunk, const mw_strides* strides,
                              mw_stream_t stream) {
  const char* fn = "mw_kvcache_append";
  int st = check_cache(fn, c);
  if (st) return st;
  st = check_ptrs(fn, {{"k_chunk", k_chunk}, {"v_chunk", v_chunk}});
  if (st) return st;
  if (strides != nullptr) {
    st = check_view(fn, "k_chunk", strides[0], c->B, c->H, c->L, c->D, false);
    if (st) return st;
    st = check_view(fn, "v_chunk", strides[1], c->B, c->H, c->L, c->D, false);
    if (st) return st;
  }
  if (c->head - c->tail == c->S) return fail(MW_EFULL, "%s: all %d slots hold live chunks; evict first", fn, c->S);
  const long long n = (long long)c->B * c->H * c->L * c->D;
  const int slot = (int)(c->head % c->S);
  if (c->elem_bytes == 1) {  // quantize into the e4m3 slot
    const mw::Strides cs = contiguous(c->H, c->L, c->D);
    mw::QuantJobs jobs{};
    jobs.j[0] = {static_cast<const uint16_t*>(k_chunk), strides ? to_internal(strides[0]) : cs,
                 static_cast<uint8_t*>(c->k_slots) + (long long)slot * n, 1.f / c->k_scale};
    jobs.j[1] = {static_cast<const uint16_t*>(v_chunk), strides ? to_internal(strides[1]) : cs,
                 static_cast<uint8_t*>(c->v_slots) + (long long)slot * n, 1.f / c->v_scale};
    hipError_t e = mw::launch_quantize_fp8(jobs, 2, c->B, c->H, c->L, c->D, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_status(fn, e);
    c->rope_at_commit[slot] = c->rope_total;  // shifts from here on are pending for this chunk
    c->head += 1;
    return ok();
  }
  uint16_t* kd = static_cast<uint16_t*>(c->k_slots) + (long long)slot * n;
  uint16_t* vd = static_cast<uint16_t*>(c->v_slots) + (long long)slot * n;
  const uint16_t* ks = static_cast<const uint16_t*>(k_chunk);
  const uint16_t* vs = static_cast<const uint16_t*>(v_chunk);
  const mw::Strides cs = contiguous(c->H, c->L, c->D);
  const bool dense = strides == nullptr ||
                     (strides[0].b == cs.b && strides[0].h == cs.h && strides[0].t == cs.t && strides[1].b == cs.b &&
                      strides[1].h == cs.h && strides[1].t == cs.t);
  hipError_t e = dense ? mw::launch_kv_copy(ks, vs, kd, vd, n, static_cast<hipStream_t>(stream))
                       : mw::launch_kv_gather(ks, vs, to_internal(strides[0]), to_internal(strides[1]), kd, vd, c->B,
                                              c->H, c->L, c->D, static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return hip_status(fn, e);
  c->head += 1;
  return ok();
}

int mw_kvcache_append(mw_kvcache* c, const void* k_chunk, const void* v_chunk, mw_stream_t stream) {
  return mw_kvcache_append_strided(c, k_chunk, v_chunk, nullptr, stream);
}

int mw_kvcache_set_sink(mw_kvcache* c, const void* k_sink, const void* v_sink, int sink_len) {
  const char* fn = "mw_kvcache_set_sink";
  int st = check_cache(fn, c);
  if (st) return st;
  if (sink_len < 0) return fail(MW_EINVAL, "%s: sink_len must be >= 0", fn);
  if (sink_len == 0) {
    c->k_sink = nullptr;
    c->v_sink = nullptr;
    c->sink_len = 0;
    return ok();
  }
  st = check_ptrs(fn, {{"k_sink", k_sink}, {"v_sink", v_sink}});
  if (st) return st;
  if (sink_len > kMaxT / 2) return fail(MW_EUNSUPPORTED, "%s: sink_len %d too large", fn, sink_len);
  c->k_sink = k_sink;
  c->v_sink = v_sink;
  c->sink_len = sink_len;
  return ok();
}

int mw_kvcache_rope_shift(mw_kvcache* c, int shift, const mw_rope* rope, mw_stream_t stream) {
  const char* fn = "mw_kvcache_rope_shift";
  int st = check_cache(fn, c);
  if (st) return st;
  if (rope == nullptr) return fail(MW_EINVAL, "%s: rope is NULL", fn);
  st = check_band(fn, rope, c->D);
  if (st) return st;
  if (c->elem_bytes == 1) {
    // e4m3 slots: rotation on load; record the shift (and the band of the first)
    if (c->rope_set && (rope->dim_offset != c->rope_offset || rope->dim_count != c->rope_count ||
                        rope->theta != c->rope_theta))
      return fail(MW_EINVAL, "%s: the band of this e4m3 cache's shifts is [%d, %d) with theta %g; got [%d, %d), %g", fn,
                  c->rope_offset, c->rope_offset + c->rope_count, (double)c->rope_theta, rope->dim_offset,
                  rope->dim_offset + rope->dim_count, (double)rope->theta);
    c->rope_offset = rope->dim_offset;
    c->rope_count = rope->dim_count;
    c->rope_theta = rope->theta;
    c->rope_set = 1;
    c->rope_total += shift;
    return ok();
  }
  const long long live = c->head - c->tail;
  if (shift == 0 || live == 0) return ok();
  mw::RopeTable tab{};
  const int np = rope->dim_count / 2;
  for (int i = 0; i < np; ++i) {
    const double freq = std::pow((double)rope->theta, -2.0 * i / rope->dim_count);
    const double ang = -(double)shift * freq;
    tab.c[i] = (float)std::cos(ang);
    tab.s[i] = (float)std::sin(ang);
  }
  const long long rows = (long long)c->B * c->H * c->L;
  hipError_t e = mw::launch_rope_shift(static_cast<uint16_t*>(c->k_slots), rows * c->D, c->S, (int)(c->tail % c->S),
                                       (int)live, rows, c->D, rope->dim_offset, np, tab,
                                       static_cast<hipStream_t>(stream));
  return hip_status(fn, e);
}

int mw_kvcache_evict(mw_kvcache* c, int n_chunks) {
  const char* fn = "mw_kvcache_evict";
  int st = check_cache(fn, c);
  if (st) return st;
  if (n_chunks < 0) return fail(MW_EINVAL, "%s: n_chunks must be >= 0", fn);
  if (n_chunks > c->head - c->tail)
    return fail(MW_EEMPTY, "%s: cannot evict %d chunks, only %lld are live", fn, n_chunks,
                (long long)(c->head - c->tail));
  c->tail += n_chunks;
  return ok();
}

int mw_kvcache_live(const mw_kvcache* c) {
  int st = check_cache("mw_kvcache_live", c);
  if (st) return st;
  return (int)(c->head - c->tail);
}

int mw_kvcache_slot_of(const mw_kvcache* c, int64_t chunk) {
  if (c == nullptr || c->S < 1) return -1;
  if (chunk < c->tail || chunk >= c->head) return -1;
  return (int)(chunk % c->S);
}

// sustained MFMA rate assumed by the split model of the e4m3 kernel
constexpr double kFp8Flops = 1.6e15;

static long long window_chunks(const mw_kvcache* c, int window) {
  const long long live = c->head - c->tail;
  return window < 0 ? live : window;
}

// Workspace bytes of an e4m3 cache's window keys rotated on load (w chunks),
// a multiple of 256 so that the split partials after them stay aligned.
static size_t rope_window_bytes(const mw_kvcache* c, long long w) {
  const size_t b = (size_t)w * c->B * c->H * c->L * c->D;
  return (b + 255) & ~(size_t)255;
}

// Shifts pending per window chunk of an e4m3 cache (window order), and
// whether any is; the rotation on load runs only then.
static bool rope_pending(const mw_kvcache* c, long long w, long long* pend) {
  bool any = false;
  for (long long i = 0; i < w; ++i) {
    const long long chunk = c->head - w + i;
    pend[i] = c->rope_total - c->rope_at_commit[chunk % c->S];
    any = any || pend[i] != 0;
  }
  return any;
}

size_t mw_chunk_attn_cached_workspace_size(const mw_kvcache* c, int n_queued, int q_len, int window) {
  if (c == nullptr || n_queued < 1 || q_len < 1 || c->L < 1 || (c->D != 64 && c->D != 72 && c->D != 128)) return 0;
  const long long w = window_chunks(c, window);
  const long long tq = (long long)n_queued * q_len;
  const long long tk = c->sink_len + w * c->L + tq;
  if (tq > kMaxT || tk > kMaxT) return 0;
  const int bh = c->B * c->H;
  // the larger of the two visibility rules' plans (a call given less workspace
  // plans within it)
  const mw::FwdChoice ch = c->elem_bytes == 1 ? mw::fwd8_choice((int)tq) : mw::fwd_choice(c->D, true, (int)tq);
  size_t bytes = 0;
  for (const bool isolated : {false, true}) {
    const mw::SplitPlan sp =
        c->elem_bytes == 1
            ? mw::fwd_plan_splits(ch, kFp8Flops, 1, c->D, bh, (int)tq, (int)tk, q_len, isolated, (size_t)-1)
            : mw::fwd_plan_cached(c->D, bh, (int)tq, (int)tk, q_len, isolated, (size_t)-1);
    bytes = std::max(bytes, mw::fwd_split_bytes(c->D, bh, mw::fwd_split_rows(ch.bm, (int)tq, sp), sp.n_splits));
  }
  if (c->elem_bytes == 1 && w > 0) bytes += rope_window_bytes(c, w);  // keys rotated on load
  return bytes;
}

int mw_chunk_attn_cached_plan(const mw_kvcache* c, int n_queued, int q_len, int window, int flags,
                              size_t workspace_bytes, int* n_splits, int* n_whole) {
  const char* fn = "mw_chunk_attn_cached_plan";
  int st = check_cache(fn, c);
  if (st) return st;
  if (n_splits == nullptr || n_whole == nullptr) return fail(MW_EINVAL, "%s: null output pointer", fn);
  if (n_queued < 1 || q_len < 1) return fail(MW_EINVAL, "%s: n_queued and q_len must be >= 1", fn);
  if (flags != MW_QUEUED_CAUSAL && flags != MW_QUEUED_ISOLATED) return fail(MW_EINVAL, "%s: unknown flags %d", fn, flags);
  const long long live = c->head - c->tail;
  if (window < -1) return fail(MW_EINVAL, "%s: window must be >= -1", fn);
  const long long w = window_chunks(c, window);
  if (w > live) return fail(MW_EINVAL, "%s: window %d exceeds the %lld live chunks", fn, window, live);
  if (w > MW_MAX_WINDOW) return fail(MW_EUNSUPPORTED, "%s: window %lld exceeds %d", fn, w, MW_MAX_WINDOW);
  if (n_queued > MW_MAX_QUEUED) return fail(MW_EUNSUPPORTED, "%s: n_queued %d exceeds %d", fn, n_queued, MW_MAX_QUEUED);
  const long long tq = (long long)n_queued * q_len;
  const long long tk = c->sink_len + w * c->L + tq;
  if (tk > kMaxT) return fail(MW_EUNSUPPORTED, "%s: too many tokens", fn);
  const int bh = c->B * c->H;
  const bool isolated = flags == MW_QUEUED_ISOLATED;
  if (c->elem_bytes == 1) {  // the rotated window keys come first in the workspace while shifts are pending
    long long pend[MW_MAX_WINDOW];
    if (rope_pending(c, w, pend)) {
      const size_t kw = rope_window_bytes(c, w);
      workspace_bytes = workspace_bytes > kw ? workspace_bytes - kw : 0;
    }
  }
  const mw::SplitPlan sp =
      c->elem_bytes == 1
          ? mw::fwd_plan_splits(mw::fwd8_choice((int)tq), kFp8Flops, 1, c->D, bh, (int)tq, (int)tk, q_len, isolated,
                                workspace_bytes)
          : mw::fwd_plan_cached(c->D, bh, (int)tq, (int)tk, q_len, isolated, workspace_bytes);
  *n_splits = sp.n_splits;
  *n_whole = sp.n_whole;
  return MW_OK;
}

int mw_chunk_attn_cached_strided(const void* q, const void* k_new, const void* v_new, int n_queued, int q_len,
                                 const mw_kvcache* c, int window, int flags, void* o, float* lse, float scale,
                                 void* workspace, size_t workspace_bytes, const mw_strides* strides,
                                 mw_stream_t stream) {
  const char* fn = "mw_chunk_attn_cached";
  int st = check_cache(fn, c);
  if (st) return st;
  if (c->elem_bytes != 2) return fail(MW_EINVAL, "%s: the cache holds e4m3 slots (use mw_chunk_attn_cached_fp8)", fn);
  st = check_ptrs(fn, {{"q", q}, {"k_new", k_new}, {"v_new", v_new}, {"o", o}});
  if (st) return st;
  if (lse != nullptr && !aligned16(lse)) return fail(MW_EALIGN, "%s: lse is not 16-byte aligned", fn);
  if (workspace != nullptr && !aligned16(workspace)) return fail(MW_EALIGN, "%s: workspace is not 16-byte aligned", fn);
  if (n_queued < 1 || q_len < 1) return fail(MW_EINVAL, "%s: n_queued and q_len must be >= 1", fn);
  if (flags != MW_QUEUED_CAUSAL && flags != MW_QUEUED_ISOLATED) return fail(MW_EINVAL, "%s: unknown flags %d", fn, flags);
  if (!(scale > 0.f) || !std::isfinite(scale)) return fail(MW_EINVAL, "%s: scale must be finite and > 0", fn);
  const long long live = c->head - c->tail;
  if (window < -1) return fail(MW_EINVAL, "%s: window must be >= -1", fn);
  const long long w = window_chunks(c, window);
  if (w > live) return fail(MW_EINVAL, "%s: window %d exceeds the %lld live chunks", fn, window, live);
  if (w > MW_MAX_WINDOW) return fail(MW_EUNSUPPORTED, "%s: window %lld exceeds %d", fn, w, MW_MAX_WINDOW);
  if (n_queued > MW_MAX_QUEUED) return fail(MW_EUNSUPPORTED, "%s: n_queued %d exceeds %d", fn, n_queued, MW_MAX_QUEUED);
  const long long nq_tok = (long long)n_queued * q_len;
  if (nq_tok + w * c->L + c->sink_len > kMaxT) return fail(MW_EUNSUPPORTED, "%s: too many tokens", fn);
  mw::Strides sv[4];
  const char* names[4] = {"q", "k_new", "v_new", "o"};
  for (int i = 0; i < 4; ++i) {
    if (strides == nullptr) {
      sv[i] = contiguous(c->H, (int)nq_tok, c->D);
      continue;
    }
    st = check_view(fn, names[i], strides[i], c->B, c->H, (int)nq_tok, c->D, i == 3);
    if (st) return st;
    sv[i] = to_internal(strides[i]);
  }
  mw::FwdParams p{};
  p.q = static_cast<const uint16_t*>(q);
  p.k = static_cast<const uint16_t*>(k_new);
  p.v = static_cast<const uint16_t*>(v_new);
  p.o = static_cast<uint16_t*>(o);
  p.lse = lse;
  p.BH = c->B * c->H;
  p.H = c->H;
  p.Tq = (int)nq_tok;
  p.vis_mode = flags == MW_QUEUED_CAUSAL ? 1 : 2;
  p.L = c->L;
  p.sink_len = c->sink_len;
  p.k_sink = static_cast<const uint16_t*>(c->k_sink);
  p.v_sink = static_cast<const uint16_t*>(c->v_sink);
  p.wL = (int)(c->sink_len + w * c->L);
  p.Tk = p.wL + p.Tq;
  p.qlen = q_len;
  p.scale_log2 = scale * kLog2e;
  p.scale_ln = scale;
  p.k_slots = static_cast<const uint16_t*>(c->k_slots);
  p.v_slots = static_cast<const uint16_t*>(c->v_slots);
  p.slot_stride = (long long)c->B * c->H * c->L * c->D;
  p.S = c->S;
  p.first_slot = (int)((c->head - w) % c->S);
  const mw::SplitPlan sp = mw::fwd_plan_cached(c->D, p.BH, p.Tq, p.Tk, q_len, flags == MW_QUEUED_ISOLATED,
                                               workspace != nullptr ? workspace_bytes : 0);
  p.n_splits = sp.n_splits;
  p.n_whole = sp.n_whole;
  p.part = static_cast<float*>(workspace);
  p.sq = sv[0];
  p.sk = sv[1];
  p.sv = sv[2];
  p.so = sv[3];
  return hip_status(fn, mw::launch_fwd(p, c->D, true, static_cast<hipStream_t>(stream)));
}

int mw_chunk_attn_cached(const void* q, const void* k_new, const void* v_new, int n_queued, int q_len,
                         const mw_kvcache* c, int window, int flags, void* o, float* lse, float scale,
                         void* workspace, size_t workspace_bytes, mw_stream_t stream) {
  return mw_chunk_attn_cached_strided(q, k_new, v_new, n_queued, q_len, c, window, flags, o, lse, scale, workspace,
                                      workspace_bytes, nullptr, stream);
}

int mw_quantize_fp8(const void* x, const mw_strides* x_strides, void* y, int B, int H, int T, int D, float scale,
                    mw_stream_t stream) {
  const char* fn = "mw_quantize_fp8";
  int st = check_ptrs(fn, {{"x", x}, {"y", y}});
  if (st) return st;
  if (B < 1 || H < 1 || T < 1) return fail(MW_EINVAL, "%s: B, H and T must be >= 1 (got %d, %d, %d)", fn, B, H, T);
  if (D != 64 && D != 72 && D != 128)
    return fail(MW_EUNSUPPORTED, "%s: head dimension %d is not supported (64, 72 or 128)", fn, D);
  if ((long long)B * H * T > (1LL << 32)) return fail(MW_EUNSUPPORTED, "%s: too many rows", fn);
  if (!good_scale(scale)) return fail(MW_EINVAL, "%s: scale must be finite and > 0", fn);
  const float inv = 1.f / scale;
  if (!std::isfinite(inv) || inv == 0.f) return fail(MW_EINVAL, "%s: 1 / scale is not a finite non-zero fp32", fn);
  mw::Strides sx = contiguous(H, T, D);
  if (x_strides != nullptr) {
    st = check_view(fn, "x", *x_strides, B, H, T, D, false);
    if (st) return st;
    sx = to_internal(*x_strides);
  }
  mw::QuantJobs jobs{};
  jobs.j[0] = {static_cast<const uint16_t*>(x), sx, static_cast<uint8_t*>(y), inv};
  return hip_status(fn, mw::launch_quantize_fp8(jobs, 1, B, H, T, D, static_cast<hipStream_t>(stream)));
}

int mw_chunk_attn_cached_fp8(const void* q8, const void* k8_new, const void* v8_new, int n_queued, int q_len,
                             const mw_kvcache* c, int window, int flags, void* o, float* lse, float scale,
                             float q_scale, void* workspace, size_t workspace_bytes, const mw_strides* o_strides,
                             mw_stream_t stream) {
  const char* fn = "mw_chunk_attn_cached_fp8";
  int st = check_cache(fn, c);
  if (st) return st;
  if (c->elem_bytes != 1) return fail(MW_EINVAL, "%s: the cache holds bf16 slots (use mw_chunk_attn_cached)", fn);
  st = check_ptrs(fn, {{"q8", q8}, {"k8_new", k8_new}, {"v8_new", v8_new}, {"o", o}});
  if (st) return st;
  if (lse != nullptr && !aligned16(lse)) return fail(MW_EALIGN, "%s: lse is not 16-byte aligned", fn);
  if (workspace != nullptr && !aligned16(workspace)) return fail(MW_EALIGN, "%s: workspace is not 16-byte aligned", fn);
  if (n_queued < 1 || q_len < 1) return fail(MW_EINVAL, "%s: n_queued and q_len must be >= 1", fn);
  if (flags != MW_QUEUED_CAUSAL && flags != MW_QUEUED_ISOLATED) return fail(MW_EINVAL, "%s: unknown flags %d", fn, flags);
  if (!good_scale(scale)) return fail(MW_EINVAL, "%s: scale must be finite and > 0", fn);
  if (!good_scale(q_scale)) return fail(MW_EINVAL, "%s: q_scale must be finite and > 0", fn);
  const float cscale = scale * q_scale * c->k_scale * kLog2e;
  if (!(cscale > 0.f) || !std::isfinite(cscale))
    return fail(MW_EINVAL, "%s: scale * q_scale * k_scale is not a finite non-zero fp32", fn);
  const long long live = c->head - c->tail;
  if (window < -1) return fail(MW_EINVAL, "%s: window must be >= -1", fn);
  const long long w = window_chunks(c, window);
  if (w > live) return fail(MW_EINVAL, "%s: window %d exceeds the %lld live chunks", fn, window, live);
  if (w > MW_MAX_WINDOW) return fail(MW_EUNSUPPORTED, "%s: window %lld exceeds %d", fn, w, MW_MAX_WINDOW);
  if (n_queued > MW_MAX_QUEUED) return fail(MW_EUNSUPPORTED, "%s: n_queued %d exceeds %d", fn, n_queued, MW_MAX_QUEUED);
  const long long nq_tok = (long long)n_queued * q_len;
  if (nq_tok + w * c->L + c->sink_len > kMaxT) return fail(MW_EUNSUPPORTED, "%s: too many tokens", fn);
  mw::Strides so = contiguous(c->H, (int)nq_tok, c->D);
  if (o_strides != nullptr) {
    st = check_view(fn, "o", *o_strides, c->B, c->H, (int)nq_tok, c->D, true);
    if (st) return st;
    so = to_internal(*o_strides);
  }
  mw::FwdParams p{};
  p.q = static_cast<const uint16_t*>(q8);  // e4m3 bytes (see FwdParams)
  p.k = static_cast<const uint16_t*>(k8_new);
  p.v = static_cast<const uint16_t*>(v8_new);
  p.o = static_cast<uint16_t*>(o);
  p.lse = lse;
  p.BH = c->B * c->H;
  p.H = c->H;
  p.Tq = (int)nq_tok;
  p.vis_mode = flags == MW_QUEUED_CAUSAL ? 1 : 2;
  p.L = c->L;
  p.sink_len = c->sink_len;
  p.k_sink = static_cast<const uint16_t*>(c->k_sink);
  p.v_sink = static_cast<const uint16_t*>(c->v_sink);
  p.wL = (int)(c->sink_len + w * c->L);
  p.Tk = p.wL + p.Tq;
  p.qlen = q_len;
  p.scale_log2 = cscale;
  p.scale_ln = scale;
  p.k_slots = static_cast<const uint16_t*>(c->k_slots);
  p.v_slots = static_cast<const uint16_t*>(c->v_slots);
  p.slot_stride = (long long)c->B * c->H * c->L * c->D;  // bytes = elements
  p.S = c->S;
  p.first_slot = (int)((c->head - w) % c->S);
  // Rotation on load of window keys with shifts pending: the start of the
  // workspace is reserved for the rotated window (the plan never depends on
  // which of the two routes runs).  Calls with one query tile per head rotate each staged K tile
  // inside the attention kernel; the others rotate the window into the
  // reserved bytes first and the attention reads the keys from there.
  long long pend[MW_MAX_WINDOW];
  char* ws = static_cast<char*>(workspace);
  size_t ws_bytes = workspace != nullptr ? workspace_bytes : 0;
  const bool pending = rope_pending(c, w, pend);
  uint8_t* k_win = nullptr;
  if (pending) {
    const size_t kw = rope_window_bytes(c, w);
    if (ws == nullptr || ws_bytes < kw)
      return fail(MW_EINVAL, "%s: shifts are pending on the window; its rotated keys need %zu bytes of workspace, got %zu",
                  fn, kw, ws_bytes);
    k_win = reinterpret_cast<uint8_t*>(ws);
    ws += kw;
    ws_bytes -= kw;
  }
  const mw::SplitPlan sp = mw::fwd_plan_splits(mw::fwd8_choice(p.Tq), kFp8Flops, 1, c->D, p.BH, p.Tq, p.Tk, q_len,
                                               flags == MW_QUEUED_ISOLATED, ws_bytes);
  mw::RopeStage rs{};  // n_pairs = 0: nothing rotated in staging
  if (pending) {
    const int np = c->rope_count / 2;
    for (long long i = 0; i < w; ++i) rs.a.pend[i] = pend[i];
    for (int i = 0; i < np; ++i) {
      const double freq = std::pow((double)c->rope_theta, -2.0 * i / c->rope_count);
      rs.a.c1[i] = std::cos(freq);
      rs.a.s1[i] = std::sin(freq);
    }
    if (mw::fwd8_rotates_in_staging(p.Tq, p.Tk, c->L, sp)) {
      rs.n_pairs = np;
      rs.dim_offset = c->rope_offset;
    } else {
      hipError_t e = mw::launch_rope_load_fp8(static_cast<const uint8_t*>(c->k_slots), k_win, p.slot_stride, c->S,
                                              p.first_slot, (int)w, (long long)c->B * c->H * c->L, c->rope_offset, np,
                                              rs.a, static_cast<hipStream_t>(stream));
      if (e != hipSuccess) return hip_status(fn, e);
      p.k_win = k_win;
    }
  }
  p.n_splits = sp.n_splits;
  p.n_whole = sp.n_whole;
  p.part = reinterpret_cast<float*>(ws_bytes > 0 ? ws : nullptr);
  p.so = so;
  p.o_scale = c->v_scale;
  return hip_status(fn, mw::launch_fwd_fp8(p, rs, static_cast<hipStream_t>(stream)));
}

}  // extern "C"
