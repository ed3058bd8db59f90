// Kernel parameter blocks and launchers (host <-> device interface inside the library).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mw {

// Forward / cached attention.  Queries: [BH, Tq, D]; keys: the (virtual) key
// sequence of length vis.Tk described below; output O [BH, Tq, D], lse [BH, Tq].
struct FwdParams {
  const uint16_t* q;
  const uint16_t* k;  // training: [BH, Tk, D]; cached: the queued chunks' keys [BH, Tq, D]
  const uint16_t* v;
  uint16_t* o;
  float* lse;  // may be null (cached attention)
  int BH;
  int Tq;
  int n_qtiles;   // set by the launcher from its tile configuration
  int vis_mode;  // VisMode
  int L;         // chunk length (training) / committed chunk length (cached)
  int Tk;        // keys in the (virtual) sequence
  int qlen;      // queued chunk length (cached)
  int wL;        // window tokens = n_window * L (cached; 0 in training)
  float scale_log2;  // softmax scale * log2(e)
  float scale_ln;    // unused by the kernels; kept for the host's records
  // cached attention only: the window lives in ring slots
  const uint16_t* k_slots;
  const uint16_t* v_slots;
  long long slot_stride;  // elements per slot (B*H*L*D)
  int S;                  // ring capacity in slots
  int first_slot;         // slot of the oldest window chunk; chunk i of the window is in slot (first_slot+i)%S
};

struct BwdParams {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  const uint16_t* o;
  const uint16_t* d_o;
  const float* lse;
  float* delta;  // workspace [BH, T]: rowsum(dO * O)
  float* lse2;   // workspace [BH, T]: LSE * log2(e)
  uint16_t* dq;
  uint16_t* dk;
  uint16_t* dv;
  int BH;
  int T;
  int L;
  float scale;
  float scale_log2;
};

// Tile sizes (shared with the host for grid computation).
constexpr int DKV_BN = 128;   // keys per workgroup in the dK/dV kernel
constexpr int DKV_BM = 64;    // queries per step in the dK/dV kernel
constexpr int DQ_BM = 128;    // queries per workgroup in the dQ kernel
constexpr int DQ_BN = 64;     // keys per step in the dQ kernel

hipError_t launch_fwd(const FwdParams& p, int D, bool cached, hipStream_t stream);
hipError_t launch_bwd(const BwdParams& p, int D, hipStream_t stream);
hipError_t launch_kv_copy(const uint16_t* k_src, const uint16_t* v_src, uint16_t* k_dst,
                          uint16_t* v_dst, long long n_elems, hipStream_t stream);

}  // namespace mw
