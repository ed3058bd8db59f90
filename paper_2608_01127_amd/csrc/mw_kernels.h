// Kernel parameter blocks and launchers (host <-> device interface inside the library).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mw {

// Element strides of a [B, H, T, D] tensor view (D contiguous): element
// (b, h, t, d) is at base + b * b_ + h * h_ + t * t_ + d.
struct Strides {
  long long b;
  long long h;
  long long t;
};

// Forward / cached attention.  Queries: [BH, Tq, D]; keys: the (virtual) key
// sequence of length vis.Tk described below; output O [BH, Tq, D], lse [BH, Tq].
struct FwdParams {
  const uint16_t* q;
  const uint16_t* k;  // training: [BH, Tk, D]; cached: the queued chunks' keys [BH, Tq, D]
  const uint16_t* v;
  uint16_t* o;
  float* lse;  // may be null (cached attention)
  int BH;
  int H;
  int Tq;
  int n_qtiles;   // set by the launcher from its tile configuration
  int vis_mode;  // VisMode
  int L;         // chunk length (training) / committed chunk length (cached)
  int Tk;        // keys in the (virtual) sequence
  int qlen;      // queued chunk length (cached)
  int wL;        // history tokens = sink_len + n_window * L (cached; 0 in training)
  float scale_log2;  // softmax scale * log2(e)
  float scale_ln;    // unused by the kernels; kept for the host's records
  // cached attention only: the window lives in ring slots
  const uint16_t* k_slots;
  const uint16_t* v_slots;
  const uint16_t* k_sink;  // [BH, sink_len, D], first in the key sequence
  const uint16_t* v_sink;
  int sink_len;
  long long slot_stride;  // elements per slot (B*H*L*D)
  int S;                  // ring capacity in slots
  int first_slot;         // slot of the oldest window chunk; chunk i of the window is in slot (first_slot+i)%S
  // key-range splitting (cached attention, n_splits > 1): the n_whole heaviest
  // (last) query tiles of each head run unsplit; each of the others is covered
  // by n_splits workgroups, one per 1/n_splits of its key tiles, which write
  // fp32 partials for a merge kernel (see attn_fwd.hip).  The split tiles are a
  // head's first ones: rows [0, split_rows), set by the launcher.
  int n_splits;
  int n_whole;
  int split_rows;
  float* part;  // [n_splits][BH][split_rows][D] unnormalised O, then [n_splits][BH][split_rows][2] (m, l)
  // views of q, k (training keys / queued keys), v and o; lse and the ring
  // are always contiguous
  Strides sq, sk, sv, so;
  // fp8 kernel only: q, k, v, the slots and the sink hold e4m3 bytes
  // (contiguous; element strides are byte strides) and O is multiplied by
  // o_scale (the V scale) before it is stored
  float o_scale;
  // fp8 kernel only: window keys rotated on load, [n_window][BH, L, 128] bytes
  // in window order (chunk w at w * slot_stride), or null (keys from the slots)
  const uint8_t* k_win;
};

struct BwdParams {
  const uint16_t* q;
  const uint16_t* k;
  const uint16_t* v;
  const uint16_t* o;
  const uint16_t* d_o;
  const float* lse;
  float* delta;  // workspace [BH, T]: -rowsum(dO * O)
  float* lse2;   // workspace [BH, T]: LSE * log2(e)
  uint16_t* dq;
  uint16_t* dk;
  uint16_t* dv;
  int BH;
  int H;
  int T;
  int L;
  float scale;
  float scale_log2;
  // views of the [B, H, T, D] tensors; lse, delta and lse2 are contiguous [B, H, T]
  Strides sq, sk, sv, so, sdo, sdq, sdk, sdv;
};


hipError_t launch_fwd_64(const FwdParams& p, bool cached, hipStream_t stream);
hipError_t launch_fwd_72(const FwdParams& p, bool cached, hipStream_t stream);
hipError_t launch_fwd_128(const FwdParams& p, bool cached, hipStream_t stream);
// cached attention at D = 128: the 256-row configuration, and the ones with
// `bm` (64 or 128) query rows per workgroup
hipError_t launch_fwd_cached_128(const FwdParams& p, hipStream_t stream);
hipError_t launch_fwd_decode_128(const FwdParams& p, int bm, hipStream_t stream);
inline hipError_t launch_fwd(const FwdParams& p, int D, bool cached, hipStream_t stream) {
  return D == 64 ? launch_fwd_64(p, cached, stream)
                 : (D == 72 ? launch_fwd_72(p, cached, stream) : launch_fwd_128(p, cached, stream));
}
// Workgroups per CU that the forward kernel of each unit holds at once
// (runtime occupancy; the value the kernels' register and LDS use gives as
// built where no device is present): the training or cached kernel of
// launch_fwd_64 / _72 / _128, and the few-rows kernel of `bm` rows.
int fwd_resident_wgs_64(bool cached);
int fwd_resident_wgs_72(bool cached);
int fwd_resident_wgs_128(bool cached);
int fwd_resident_wgs_cached_128();
int fwd_resident_wgs_decode_128(int bm);
// Query rows per workgroup, keys per main-loop step and resident workgroups
// per CU of the tile configuration the forward launcher picks for a shape.
struct FwdChoice {
  int bm;
  int bk;
  int wg_per_cu;
};
FwdChoice fwd_choice(int D, bool cached, int Tq);
// fp8 (e4m3) cached attention at D = 128: its tile configuration and launcher
// (FwdParams as described above), and the merge of split partials (D = 128).
FwdChoice fwd8_choice(int Tq);
hipError_t launch_combine(const FwdParams& p, int D, hipStream_t stream);
// bf16 view -> contiguous e4m3, code = RNE(clamp(x * inv_scale, +-448)); up to
// two jobs of the same shape in one launch.
struct QuantJob {
  const uint16_t* x;
  Strides sx;
  uint8_t* y;
  float inv_scale;
};
struct QuantJobs {
  QuantJob j[2];
};
hipError_t launch_quantize_fp8(const QuantJobs& jobs, int n_jobs, int B, int H, int T, int D, hipStream_t stream);
// Key-range split plan of a cached call: the n_whole heaviest query tiles of
// each head run unsplit, the others over n_splits key ranges (n_splits = 1:
// no split, n_whole = 0).
struct SplitPlan {
  int n_splits;
  int n_whole;
};
// Plan for a call run by the configuration `ch` at `flops` FLOP/s of
// sustained MFMA throughput, over K/V elements of `kv_bytes` bytes, with
// queued chunks of `qlen` rows (`isolated`: each sees only the history and
// itself), within `ws_bytes` of workspace.
SplitPlan fwd_plan_splits(const FwdChoice& ch, double flops, int kv_bytes, int D, int BH, int Tq, int Tk, int qlen,
                          bool isolated, size_t ws_bytes);
// The plan of the bf16 cached launcher (its configuration and sustained rate).
SplitPlan fwd_plan_cached(int D, int BH, int Tq, int Tk, int qlen, bool isolated, size_t ws_bytes);
// Rows per head covered by the split tiles (0 without a split), and the
// workspace bytes of their partials.
int fwd_split_rows(int bm, int Tq, const SplitPlan& sp);
size_t fwd_split_bytes(int D, int BH, int split_rows, int n_splits);
// Grid of a forward launch with `bm`-row tiles, after setting the split fields
// of p: n_qtiles, and for a split (cached attention only) the whole-tile count
// clamped to the tiles and the rows of the split tiles.
inline long long fwd_prepare(FwdParams& p, int bm, bool cached) {
  p.n_qtiles = (p.Tq + bm - 1) / bm;
  if (p.n_splits < 1 || !cached) p.n_splits = 1;
  p.n_whole = p.n_whole < 0 ? 0 : (p.n_whole > p.n_qtiles ? p.n_qtiles : p.n_whole);
  if (p.n_whole == p.n_qtiles) p.n_splits = 1;
  if (p.n_splits == 1) p.n_whole = 0;
  p.split_rows = fwd_split_rows(bm, p.Tq, SplitPlan{p.n_splits, p.n_whole});
  return (long long)p.BH * (p.n_whole + (long long)(p.n_qtiles - p.n_whole) * p.n_splits);
}
hipError_t launch_bwd_64(const BwdParams& p, hipStream_t stream);
hipError_t launch_bwd_72(const BwdParams& p, hipStream_t stream);
hipError_t launch_bwd_128(const BwdParams& p, hipStream_t stream);
// cos/sin of the re-shift angle of each rope pair
struct RopeTable {
  float c[64];
  float s[64];
};
hipError_t launch_rope_shift(uint16_t* k_slots, long long slot_stride, int S, int first_slot, int n_live,
                             long long rows_per_slot, int D, int dim_offset, int n_pairs, const RopeTable& tab,
                             hipStream_t stream);
// Rotation on load of an e4m3 cache's window keys: window chunk w (in window
// order, in slot (first_slot + w) % S) is rotated by -pend[w] positions on the
// band [dim_offset, dim_offset + 2 n_pairs); c1[i], s1[i] are the cos and sin
// of pair i's frequency (its rotation per position).
struct RopeLoadArgs {
  long long pend[64];
  double c1[64];
  double s1[64];
};
// The same rotation done inside the e4m3 attention kernel's staging, on each
// staged K tile in LDS (calls with one query tile per head): pend[w] for the
// window chunks of the call, band as above; n_pairs = 0 rotates nothing.
struct RopeStage {
  RopeLoadArgs a;
  int n_pairs;
  int dim_offset;
};
// Window chunks one workgroup of the in-staging rotation can span (their
// cos/sin tables live in LDS).
constexpr int kRopeStageChunks = 8;
// Whether a call (Tq queued rows over Tk keys, window chunks of L keys, split
// plan sp) has one query tile per head and every workgroup's key range
// spans at most kRopeStageChunks window chunks, with chunks of at least half
// a staged tile, so that it can rotate its window keys in staging instead of
// in a separate pass.
bool fwd8_rotates_in_staging(int Tq, int Tk, int L, const SplitPlan& sp);
hipError_t launch_fwd_fp8(FwdParams p, const RopeStage& rs, hipStream_t stream);
hipError_t launch_rope_load_fp8(const uint8_t* k_slots, uint8_t* k_win, long long slot_bytes, int S, int first_slot,
                                int n_window, long long rows_per_slot, int dim_offset, int n_pairs,
                                const RopeLoadArgs& args, hipStream_t stream);
hipError_t launch_kv_copy(const uint16_t* k_src, const uint16_t* v_src, uint16_t* k_dst,
                          uint16_t* v_dst, long long n_elems, hipStream_t stream);
// Gather of a strided [B, H, L, D] K/V chunk into a contiguous slot.
hipError_t launch_kv_gather(const uint16_t* k_src, const uint16_t* v_src, Strides sk, Strides sv, uint16_t* k_dst,
                            uint16_t* v_dst, int B, int H, int L, int D, hipStream_t stream);

// Record the calling thread's status message (what mw_last_error returns)
// and return `code`; MW_OK clears it.
int set_error(int code, const char* msg);

}  // namespace mw
