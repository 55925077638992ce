// Online SLO-aware batching invoker (tg_slo_replay).
//
// Tangram's scheduler does not batch a fixed number of requests: it keeps stitching
// arriving patches onto canvases and invokes the detector function when waiting any
// longer would miss the earliest deadline in the queue (Sec. III-C, Online SLO-aware
// Batching Invoker and Alg. 2). The Latency Estimator prices a batch of b canvases at
// its profiled mean plus three standard deviations (Sec. III-C, Latency Estimator).
//
// Alg. 2 re-solves the packing of the whole queue on every arrival. With a packer that
// places patches in arrival order, a placement depends only on the patches before it,
// so the queue's packing grows by exactly one placement per arrival: this replay keeps
// one packer per queue and places each arrival once (O(1) placements per arrival
// instead of O(queue)). The host-only translation unit makes no HIP call.
#include <cmath>
#include <cstdint>
#include <new>
#include <vector>

#include "packers.h"
#include "tg.h"

namespace {

using tg_detail::GuillotinePacker;
using tg_detail::ShelfPacker;

struct Estimator {
  const double *mean;
  const double *sd;
  // Conservative inference time of b >= 1 canvases.
  double slack(int32_t b) const { return mean[b - 1] + 3.0 * sd[b - 1]; }
};

template <class Packer>
class Replay {
 public:
  Replay(const tg_slo_patch *patches, const tg_slo_params &p, int32_t *order, tg_place *place,
         tg_invocation *inv)
      : pt_(patches), p_(p), est_{p.lat_mean, p.lat_std}, order_(order), place_(place),
        inv_(inv), packer_(p.canvas_w, p.canvas_h) {}

  int32_t run(int32_t n) {
    for (int32_t i = 0; i < n; ++i) arrive(i);
    if (!queue_.empty()) fire(t_remain_, TG_FIRE_DEADLINE);
    return n_inv_;
  }

 private:
  // Places patch i after the queued ones; returns the canvases the queue then needs.
  int32_t place_next(int32_t i) {
    int32_t x, y;
    const bool fresh = packer_.put(pt_[i].w, pt_[i].h, &x, &y);
    const int32_t canvas = queue_.empty() ? 0 : canvas_ + (fresh ? 1 : 0);
    place_[i] = tg_place{canvas, x, y};
    return canvas + 1;
  }

  void arrive(int32_t i) {
    const double t = pt_[i].t_arrive;
    // The clock reached t_remain before (or exactly when) this patch arrived.
    if (!queue_.empty() && t_remain_ <= t) fire(t_remain_, TG_FIRE_DEADLINE);

    int32_t canvases = place_next(i);
    double ddl = queue_.empty() ? pt_[i].t_ddl : std::fmin(t_ddl_, pt_[i].t_ddl);
    if (!queue_.empty()) {
      const bool memory = canvases > p_.max_canvases;
      if (memory || ddl - est_.slack(canvases) < t) {
        // Invoke the queue as it was before this patch; the patch opens a new queue.
        fire(t, memory ? TG_FIRE_MEMORY : TG_FIRE_SLO);
        canvases = place_next(i);
        ddl = pt_[i].t_ddl;
      }
    }
    queue_.push_back(i);
    canvas_ = canvases - 1;
    t_ddl_ = ddl;
    t_remain_ = ddl - est_.slack(canvases);
    if (t_remain_ <= t) fire(t, TG_FIRE_DEADLINE);  // already due: invoke now
  }

  void fire(double t, int32_t reason) {
    tg_invocation &v = inv_[n_inv_++];
    v.t_fire = t;
    v.t_ddl = t_ddl_;
    v.t_slack = est_.slack(canvas_ + 1);
    v.first = emitted_;
    v.count = static_cast<int32_t>(queue_.size());
    v.n_canvases = canvas_ + 1;
    v.reason = reason;
    for (int32_t id : queue_) order_[emitted_++] = id;
    queue_.clear();
    packer_ = Packer(p_.canvas_w, p_.canvas_h);
  }

  const tg_slo_patch *pt_;
  const tg_slo_params &p_;
  Estimator est_;
  int32_t *order_;
  tg_place *place_;
  tg_invocation *inv_;
  Packer packer_;
  std::vector<int32_t> queue_;
  int32_t canvas_ = 0;  // canvas of the queue's last placement
  double t_ddl_ = 0.0;  // earliest deadline in the queue
  double t_remain_ = 0.0;
  int32_t n_inv_ = 0;
  int32_t emitted_ = 0;
};

int check(const tg_slo_patch *pt, int32_t n, const tg_slo_params &p, int32_t *bad) {
  if (p.canvas_w < 1 || p.canvas_h < 1 || p.max_canvases < 1 || p.n_lat < p.max_canvases ||
      !p.lat_mean || !p.lat_std)
    return TG_E_INVAL;
  if (p.policy != TG_PACK_GUILLOTINE_BSSF && p.policy != TG_PACK_SHELF_ARRIVAL)
    return TG_E_INVAL;
  for (int32_t b = 0; b < p.n_lat; ++b)
    if (!std::isfinite(p.lat_mean[b]) || !std::isfinite(p.lat_std[b])) return TG_E_INVAL;
  for (int32_t i = 0; i < n; ++i) {
    int code = TG_OK;
    if (pt[i].w < 1 || pt[i].h < 1 || !std::isfinite(pt[i].t_arrive) ||
        !std::isfinite(pt[i].t_ddl) || (i > 0 && pt[i].t_arrive < pt[i - 1].t_arrive))
      code = TG_E_INVAL;
    else if (pt[i].w > p.canvas_w || pt[i].h > p.canvas_h)
      code = TG_E_ROI_TOO_LARGE;
    if (code != TG_OK) {
      *bad = i;
      return code;
    }
  }
  return TG_OK;
}

}  // namespace

extern "C" int tg_slo_replay(const tg_slo_patch *patches, int32_t n, const tg_slo_params *params,
                             int32_t *order, tg_place *place, tg_invocation *inv, int32_t *n_inv,
                             int32_t *bad_index) {
  if (!params || !n_inv || !bad_index || n < 0) return TG_E_INVAL;
  if (n > 0 && (!patches || !order || !place || !inv)) return TG_E_INVAL;
  *bad_index = -1;
  *n_inv = 0;
  const tg_slo_params p = *params;
  if (int rc = check(patches, n, p, bad_index); rc != TG_OK) return rc;
  try {
    if (p.policy == TG_PACK_GUILLOTINE_BSSF) {
      Replay<GuillotinePacker> r(patches, p, order, place, inv);
      *n_inv = r.run(n);
    } else {
      Replay<ShelfPacker> r(patches, p, order, place, inv);
      *n_inv = r.run(n);
    }
    return TG_OK;
  } catch (const std::bad_alloc &) {
    return TG_E_INTERNAL;
  } catch (...) {
    return TG_E_INTERNAL;
  }
}
