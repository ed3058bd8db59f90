// Planning of the pipelined streaming denoiser (declared in include/mw.h):
// host-only arithmetic, closed form per tick.
//
// Chunk i enters the active window at tick e(i) = floor(i / stride) at
// tau = 1 and is updated once per tick for U = floor(window / stride) ticks;
// before its k-th update (k = t - e(i)) it is at tau = g(k / U) with
// g(x) = shift(1 - x) and shift(t) = s t / (1 + (s - 1) t), so the last update
// lands on tau = 0 and the chunk is committed after tick e(i) + U - 1.  Chunks
// in flight at tick t are [max(0, (t - U + 1) stride), min(N, (t + 1) stride)).
// The FIFO keeps the newest cache_chunks committed chunks, so after tick t it
// holds min(C, committed(t + 1)) of them, committed(t) = clamp((t - U + 1)
// stride, 0, N) being the chunks committed before tick t.
#include <algorithm>
#include <cmath>

#include "mw.h"
#include "mw_kernels.h"

namespace {

long long clampll(long long x, long long lo, long long hi) { return x < lo ? lo : (x > hi ? hi : x); }

int bad(const char* what) { return mw::set_error(MW_EINVAL, what); }

int validate(const mw_sched_config* c) {
  if (c == nullptr) return bad("mw_sched: config is NULL");
  if (c->window < 1 || c->window > MW_MAX_QUEUED) return bad("mw_sched: window must be 1..MW_MAX_QUEUED");
  if (c->stride < 1 || c->stride > c->window) return bad("mw_sched: stride must be 1..window");
  if (c->n_chunks < 1) return bad("mw_sched: n_chunks must be >= 1");
  if (c->cache_chunks < 0) return bad("mw_sched: cache_chunks must be >= 0");
  if (c->frames_per_chunk < 1) return bad("mw_sched: frames_per_chunk must be >= 1");
  if (c->sink_frames < 0) return bad("mw_sched: sink_frames must be >= 0");
  if (!(c->shift > 0.0) || !std::isfinite(c->shift)) return bad("mw_sched: shift must be finite and > 0");
  if (c->n_bins < 0) return bad("mw_sched: n_bins must be >= 0");
  if ((long long)c->cache_chunks * c->frames_per_chunk + c->sink_frames +
          (long long)c->window * c->frames_per_chunk > (1LL << 30))
    return mw::set_error(MW_EUNSUPPORTED, "mw_sched: positions exceed 2^30 frames");
  return MW_OK;
}

double level(long long k, long long U, double s, int n_bins) {
  const double x = 1.0 - (double)k / (double)U;
  double tau = s * x / (1.0 + (s - 1.0) * x);
  if (n_bins > 0) tau = std::nearbyint(tau * n_bins) / n_bins;
  return tau;
}

}  // namespace

extern "C" {

int64_t mw_sched_num_ticks(const mw_sched_config* cfg) {
  const int st = validate(cfg);
  if (st) return st;
  const long long U = cfg->window / cfg->stride;
  return (long long)((cfg->n_chunks - 1) / cfg->stride) + U;
}

int mw_sched_plan(const mw_sched_config* cfg, int64_t tick, mw_sched_tick* out) {
  const int st = validate(cfg);
  if (st) return st;
  if (out == nullptr) return bad("mw_sched_plan: out is NULL");
  const long long N = cfg->n_chunks, r = cfg->stride, U = cfg->window / cfg->stride, C = cfg->cache_chunks;
  const long long ticks = (N - 1) / r + U;
  if (tick < 0 || tick >= ticks) return mw::set_error(MW_EEMPTY, "mw_sched_plan: tick out of range");
  const long long t = tick;
  auto committed_before = [&](long long tt) { return clampll((tt - U + 1) * r, 0, N); };
  const long long first = committed_before(t);  // oldest in-flight chunk
  const long long last = std::min(N, (t + 1) * r);
  const long long cb = committed_before(t), ca = committed_before(t + 1);
  const long long live_before = std::min(C, cb), live_after = std::min(C, ca);
  out->tick = tick;
  out->first = (int)first;
  out->n_active = (int)(last - first);
  out->updates_per_chunk = (int)U;
  for (long long i = first; i < last; ++i) {
    const long long k = t - i / r;  // updates already made
    const double a = level(k, U, cfg->shift, cfg->n_bins), b = level(k + 1, U, cfg->shift, cfg->n_bins);
    out->tau[i - first] = a;
    out->dtau[i - first] = b - a;
  }
  for (long long i = last - first; i < MW_MAX_QUEUED; ++i) {
    out->tau[i] = 0.0;
    out->dtau[i] = 0.0;
  }
  out->n_commit = (int)(ca - cb);
  out->n_evict = (int)(live_before + (ca - cb) - live_after);
  out->rope_shift = out->n_evict * cfg->frames_per_chunk;
  out->cache_live = (int)live_after;
  out->pos_first = (int)(cfg->sink_frames + live_before * cfg->frames_per_chunk);
  return mw::set_error(MW_OK, "");
}

}  // extern "C"
