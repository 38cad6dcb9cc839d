// Host runtime of the sync-group worker entry points (include/edit_outer.h,
// "one worker of a sync group on its own GPU").
//
// A group handle owns, per sync unit, the rank's device record (its EMA pair
// and the group's last decision), the partial sums of its two norm passes
// and a completion event.  Every call validates its arguments, enqueues its
// kernels on the caller's stream and returns; the collectives between the
// calls are the caller's.
#include <algorithm>
#include <climits>
#include <cmath>
#include <cstring>
#include <new>
#include <string>
#include <vector>

#include "edit_group_internal.h"

using namespace edit;

namespace {

#define GROUP_TRY(expr)                \
  do {                                 \
    const edit_status_t st_ = (expr);  \
    if (st_ != EDIT_OK) return st_;    \
  } while (0)

edit_status_t gfail(edit_status_t s, const std::string& msg) { return set_error(s, msg.c_str()); }

edit_status_t gfail_hip(hipError_t e, const char* what) {
  return gfail(EDIT_EHIP, std::string(what) + ": " + hipGetErrorString(e));
}

int64_t gceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

struct GUnit {
  int64_t n = 0;
  int rows_norm = 1;   // blocks (= partials) of the norm pass
  int rows_dbar = 1;   // blocks (= partials) of the Delta_bar pass
  int blocks_up = 1;   // blocks of the update pass
  int blocks_clear = 1;  // blocks of the decision launch (which clears a flagged export)
  double* part_norm = nullptr;
  double* part_dbar = nullptr;
  GroupRecord* rec = nullptr;
  hipEvent_t done = nullptr;
  bool pending = false;     // `done` marks the unit's last edit_group_apply
  bool unrecorded = false;  // a norm or weights call was enqueued after it
  bool has_state = false;
};

struct Range {
  uintptr_t lo, hi;
};

bool overlap(const Range& a, const Range& b) { return a.lo < b.hi && b.lo < a.hi; }

Range range(const void* p, int64_t bytes) {
  const uintptr_t a = reinterpret_cast<uintptr_t>(p);
  return {a, a + static_cast<uintptr_t>(bytes)};
}

}  // namespace

struct edit_group {
  edit_outer_config_t cfg{};
  std::vector<int64_t> numel;
  int rank = 0;
  int device = 0;
  char* arena = nullptr;
  std::vector<GUnit> units;
};

namespace {

void destroy_group_units(edit_group* h) {
  for (GUnit& u : h->units)
    if (u.done) (void)hipEventDestroy(u.done);
  h->units.clear();
  if (h->arena) (void)hipFree(h->arena);
  h->arena = nullptr;
}

edit_status_t check_group_device(const edit_group* h) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return gfail_hip(e, "hipGetDevice");
  if (dev != h->device)
    return gfail(EDIT_EINVAL, "call made with device " + std::to_string(dev) +
                                  " current; the handle belongs to device " + std::to_string(h->device));
  return EDIT_OK;
}

edit_status_t check_layer(const edit_group* h, int32_t layer) {
  if (layer < 0 || layer >= h->cfg.num_layers)
    return gfail(EDIT_EINVAL, "layer " + std::to_string(layer) + " out of range");
  return EDIT_OK;
}

// A tensor argument of `n` elements: non-NULL and 16-byte aligned (nothing
// is required of an empty unit's pointers).
edit_status_t check_tensor(const void* p, int64_t n, const char* name) {
  if (n == 0) return EDIT_OK;
  if (!p) return gfail(EDIT_EINVAL, std::string(name) + " must not be NULL");
  if (reinterpret_cast<uintptr_t>(p) & 15u) return gfail(EDIT_EINVAL, std::string(name) + " must be 16-byte aligned");
  return EDIT_OK;
}

// A small fp64 argument: non-NULL and 8-byte aligned.
edit_status_t check_scalars(const void* p, const char* name) {
  if (!p) return gfail(EDIT_EINVAL, std::string(name) + " must not be NULL");
  if (reinterpret_cast<uintptr_t>(p) & 7u) return gfail(EDIT_EINVAL, std::string(name) + " must be 8-byte aligned");
  return EDIT_OK;
}

edit_status_t check_disjoint(const Range* r, int count, const char* what) {
  for (int a = 0; a < count; ++a)
    for (int b = a + 1; b < count; ++b)
      if (r[a].hi > r[a].lo && r[b].hi > r[b].lo && overlap(r[a], r[b])) return gfail(EDIT_EINVAL, what);
  return EDIT_OK;
}

GroupParams group_params(const edit_group* h) {
  GroupParams p;
  p.alpha = h->cfg.ema_alpha;
  p.delta = h->cfg.z_threshold;
  p.phi = h->cfg.clip_threshold;
  p.eps = h->cfg.clip_eps;
  p.warmup = h->cfg.ema_warmup_rounds;
  p.flags = h->cfg.flags;
  return p;
}

// Only the last call of a step (edit_group_apply) records the unit's
// completion event: an event record costs a few microseconds of stream time.
edit_status_t record_done(edit_group* h, int32_t layer, hipStream_t s) {
  GUnit& u = h->units[layer];
  const hipError_t e = hipEventRecord(u.done, s);
  if (e != hipSuccess) return gfail_hip(e, "hipEventRecord");
  u.pending = true;
  u.unrecorded = false;
  return EDIT_OK;
}

// Wait for the unit's enqueued work, then copy its record to the host.  After
// a norm or weights call that no apply has followed yet there is no event to
// wait on, so the whole device is synchronised instead.
edit_status_t wait_and_read(edit_group* h, int32_t layer, GroupRecord* rec) {
  GUnit& u = h->units[layer];
  hipError_t e = hipSuccess;
  if (u.unrecorded) {
    if ((e = hipDeviceSynchronize()) != hipSuccess) return gfail_hip(e, "hipDeviceSynchronize");
  } else if (u.pending && (e = hipEventSynchronize(u.done)) != hipSuccess) {
    return gfail_hip(e, "hipEventSynchronize");
  }
  if ((e = hipMemcpy(rec, u.rec, sizeof *rec, hipMemcpyDeviceToHost)) != hipSuccess)
    return gfail_hip(e, "hipMemcpy D2H");
  return EDIT_OK;
}

}  // namespace

extern "C" {

edit_status_t edit_group_init(const edit_outer_config_t* cfg, int32_t rank, edit_group_t* out) {
  if (!cfg || !out) return gfail(EDIT_EINVAL, "cfg and out must not be NULL");
  *out = nullptr;
  GROUP_TRY(validate_config(cfg));
  if (cfg->flags & EDIT_ONE_PASS) return gfail(EDIT_EINVAL, "a sync-group worker does not take EDIT_ONE_PASS");
  if (rank < 0 || rank >= cfg->num_workers)
    return gfail(EDIT_EINVAL, "rank must be in 0.." + std::to_string(cfg->num_workers - 1));
  int dev = 0, num_cu = 0;
  GROUP_TRY(current_gfx950(&dev, &num_cu));

  edit_group* h = new (std::nothrow) edit_group;
  if (!h) return gfail(EDIT_ENOMEM, "host allocation failed");
  h->cfg = *cfg;
  h->numel.assign(cfg->layer_numel, cfg->layer_numel + cfg->num_layers);
  h->cfg.layer_numel = h->numel.data();
  h->rank = rank;
  h->device = dev;
  const bool bf16 = cfg->replica_dtype == EDIT_BF16;
  const int ve = bf16 ? 8 : 4;
  const int cap_dbar = num_cu * group_dbar_blocks_per_cu();

  const size_t rec_bytes = (sizeof(GroupRecord) + 255) & ~size_t(255);
  h->units.resize(cfg->num_layers);
  std::vector<size_t> offs(cfg->num_layers);
  size_t total = 0;
  for (int l = 0; l < cfg->num_layers; ++l) {
    GUnit& u = h->units[l];
    u.n = h->numel[l];
    const int64_t nvec = u.n / ve;
    if (gceil_div(nvec, kGroupUpdateThreads) > INT32_MAX) {
      delete h;
      return gfail(EDIT_EINVAL, "layer_numel[" + std::to_string(l) + "] is too large");
    }
    u.rows_norm = static_cast<int>(std::max<int64_t>(1, gceil_div(nvec, int64_t(kGroupThreads) * kGroupNormVecs)));
    u.rows_dbar = static_cast<int>(std::max<int64_t>(1, std::min<int64_t>(cap_dbar, gceil_div(u.n / 4, kGroupThreads))));
    u.blocks_up = static_cast<int>(std::max<int64_t>(1, gceil_div(nvec, kGroupUpdateThreads)));
    u.blocks_clear = static_cast<int>(std::max<int64_t>(1, std::min<int64_t>(num_cu, gceil_div(u.n / 4, kGroupThreads))));
    offs[l] = total;
    total += rec_bytes + ((sizeof(double) * (u.rows_norm + u.rows_dbar) + 255) & ~size_t(255));
  }
  hipError_t e = hipMalloc(reinterpret_cast<void**>(&h->arena), total);
  if (e != hipSuccess) {
    h->arena = nullptr;
    destroy_group_units(h);
    delete h;
    return gfail(EDIT_ENOMEM, std::string("hipMalloc of scratch: ") + hipGetErrorString(e));
  }
  e = hipMemset(h->arena, 0, total);  // EMA pair 0, round 0
  for (int l = 0; l < cfg->num_layers && e == hipSuccess; ++l) {
    GUnit& u = h->units[l];
    u.rec = reinterpret_cast<GroupRecord*>(h->arena + offs[l]);
    u.part_norm = reinterpret_cast<double*>(h->arena + offs[l] + rec_bytes);
    u.part_dbar = u.part_norm + u.rows_norm;
    e = hipEventCreateWithFlags(&u.done, hipEventDisableTiming);
  }
  if (e == hipSuccess) e = hipDeviceSynchronize();
  if (e != hipSuccess) {
    destroy_group_units(h);
    delete h;
    return gfail_hip(e, "group init");
  }
  *out = h;
  return EDIT_OK;
}

edit_status_t edit_group_norm(edit_group_t h, int32_t layer, const float* theta, const void* replica,
                              float* delta, double* norm_out, void* stream) {
  if (!h) return gfail(EDIT_EINVAL, "NULL handle");
  GROUP_TRY(check_layer(h, layer));
  GUnit& u = h->units[layer];
  const int64_t n = u.n, rb = h->cfg.replica_dtype == EDIT_BF16 ? 2 : 4;
  GROUP_TRY(check_tensor(theta, n, "theta"));
  GROUP_TRY(check_tensor(replica, n, "replica"));
  GROUP_TRY(check_tensor(delta, n, "delta"));
  GROUP_TRY(check_scalars(norm_out, "norm_out"));
  const Range r[4] = {range(theta, 4 * n), range(replica, rb * n), range(delta, 4 * n), range(norm_out, 16)};
  GROUP_TRY(check_disjoint(r, 4, "theta, replica, delta and norm_out must not overlap"));
  GROUP_TRY(check_group_device(h));
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  const bool bf16 = h->cfg.replica_dtype == EDIT_BF16;
  hipError_t e = launch_group_norm(bf16, u.rows_norm, theta, replica, delta, n, u.part_norm, s);
  if (e == hipSuccess) e = launch_group_self(u.part_norm, u.rows_norm, u.rec, norm_out, group_params(h), s);
  if (e != hipSuccess) return gfail_hip(e, "group norm launch");
  u.has_state = true;
  u.unrecorded = true;
  return EDIT_OK;
}

edit_status_t edit_group_weights(edit_group_t h, int32_t layer, const double* gathered, double* weight_out,
                                 float* delta, void* stream) {
  if (!h) return gfail(EDIT_EINVAL, "NULL handle");
  GROUP_TRY(check_layer(h, layer));
  GUnit& u = h->units[layer];
  const int64_t n = u.n;
  const int K = h->cfg.num_workers;
  GROUP_TRY(check_scalars(gathered, "gathered"));
  GROUP_TRY(check_scalars(weight_out, "weight_out"));
  GROUP_TRY(check_tensor(delta, n, "delta"));
  const Range r[3] = {range(gathered, 16 * K), range(weight_out, 8), range(delta, 4 * n)};
  GROUP_TRY(check_disjoint(r, 3, "gathered, weight_out and delta must not overlap"));
  GROUP_TRY(check_group_device(h));
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  hipError_t e = launch_group_weights(u.blocks_clear, gathered, K, h->rank, u.rec, weight_out, delta, n,
                                      group_params(h), s);
  if (e != hipSuccess) return gfail_hip(e, "group weights launch");
  u.has_state = true;
  u.unrecorded = true;
  return EDIT_OK;
}

edit_status_t edit_group_apply(edit_group_t h, int32_t layer, const float* dbar, float* theta, float* momentum,
                               void* replica, void* stream) {
  if (!h) return gfail(EDIT_EINVAL, "NULL handle");
  GROUP_TRY(check_layer(h, layer));
  GUnit& u = h->units[layer];
  const int64_t n = u.n, rb = h->cfg.replica_dtype == EDIT_BF16 ? 2 : 4;
  GROUP_TRY(check_tensor(dbar, n, "dbar"));
  GROUP_TRY(check_tensor(theta, n, "theta"));
  GROUP_TRY(check_tensor(momentum, n, "momentum"));
  GROUP_TRY(check_tensor(replica, n, "replica"));
  const Range r[4] = {range(dbar, 4 * n), range(theta, 4 * n), range(momentum, 4 * n), range(replica, rb * n)};
  GROUP_TRY(check_disjoint(r, 4, "dbar, theta, momentum and replica must not overlap"));
  GROUP_TRY(check_group_device(h));
  hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  const bool bf16 = h->cfg.replica_dtype == EDIT_BF16;
  const GroupParams prm = group_params(h);
  hipError_t e = launch_group_dbar(u.rows_dbar, u.rec, dbar, n, u.part_dbar, s);
  if (e == hipSuccess) e = launch_group_clip(u.part_dbar, u.rows_dbar, u.rec, prm, s);
  if (e == hipSuccess && n > 0)
    e = launch_group_update(bf16, u.blocks_up, u.rec, dbar, theta, momentum, replica, n, h->cfg.outer_lr,
                            h->cfg.momentum, s);
  if (e != hipSuccess) return gfail_hip(e, "group apply launch");
  u.has_state = true;
  return record_done(h, layer, s);
}

edit_status_t edit_group_state_get(edit_group_t h, int32_t layer, edit_layer_state_t* out) {
  if (!h || !out) return gfail(EDIT_EINVAL, "NULL argument");
  GROUP_TRY(check_layer(h, layer));
  if (!h->units[layer].has_state) return gfail(EDIT_ESTATE, "unit has neither stepped nor had its state set");
  GROUP_TRY(check_group_device(h));
  GroupRecord rec;
  GROUP_TRY(wait_and_read(h, layer, &rec));
  std::memset(out, 0, sizeof *out);
  const int K = h->cfg.num_workers;
  out->round = rec.round;
  out->num_workers = K;
  out->rolled_back = rec.rollback;
  out->z_tested = rec.z_tested;
  out->ema_mean[h->rank] = rec.mu;
  out->ema_std[h->rank] = rec.sigma;
  for (int j = 0; j < K; ++j) {
    out->norm[j] = rec.norm[j];
    out->weight[j] = rec.weight[j];
    out->anomalous[j] = rec.anomalous[j];
  }
  out->synced_norm = rec.synced_norm;
  out->clip_coef = rec.clip_coef;
  return EDIT_OK;
}

edit_status_t edit_group_state_set(edit_group_t h, int32_t layer, const edit_layer_state_t* in) {
  if (!h || !in) return gfail(EDIT_EINVAL, "NULL argument");
  GROUP_TRY(check_layer(h, layer));
  if (in->round < 0) return gfail(EDIT_EINVAL, "round must be >= 0");
  const double mu = in->ema_mean[h->rank], sigma = in->ema_std[h->rank];
  if (!std::isfinite(mu) || !(sigma >= 0.0) || !std::isfinite(sigma))
    return gfail(EDIT_EINVAL, "EMA state must be finite with ema_std >= 0");
  GROUP_TRY(check_group_device(h));
  GroupRecord rec;
  GROUP_TRY(wait_and_read(h, layer, &rec));
  rec.mu = mu;
  rec.sigma = sigma;
  rec.round = in->round;
  rec.stepped = 1;
  const hipError_t e = hipMemcpy(h->units[layer].rec, &rec, sizeof rec, hipMemcpyHostToDevice);
  if (e != hipSuccess) return gfail_hip(e, "hipMemcpy H2D");
  h->units[layer].has_state = true;
  return EDIT_OK;
}

void edit_group_destroy(edit_group_t h) {
  if (!h) return;
  int prev = -1;
  if (hipGetDevice(&prev) == hipSuccess && prev != h->device) (void)hipSetDevice(h->device);
  bool unrecorded = false;
  for (GUnit& u : h->units) {
    unrecorded = unrecorded || u.unrecorded;
    if (u.pending) (void)hipEventSynchronize(u.done);
  }
  if (unrecorded) (void)hipDeviceSynchronize();
  destroy_group_units(h);
  if (prev >= 0 && prev != h->device) (void)hipSetDevice(prev);
  delete h;
}

}  // extern "C"
