// Host runtime of libedit_outer.so: the C ABI declared in include/edit_outer.h.
//
// A handle owns, per sync unit: the device record (EMA state + decision),
// the per-block Gram partials of pass 1, a completion event and (when
// profiling) four timing events.  A step validates its arguments, enqueues
// pass1 -> decide -> pass2 on the caller's stream and returns.  A round
// enqueues many units, each unit's decision folded into the next unit's
// pass-1 launch; with EDIT_ONE_PASS it enqueues one fused pass per unit and
// one record launch at the end.  The host-state round adds a staging ring
// and two copy streams.  There is no host synchronisation on the step path
// and, apart from the host-state round's copies, no host-device traffic.
#include <climits>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "edit_outer_internal.h"
#include "edit_group_internal.h"

#define EDIT_TRY(expr)                    \
  do {                                    \
    const edit_status_t st_ = (expr);     \
    if (st_ != EDIT_OK) return st_;       \
  } while (0)

using namespace edit;

namespace {

thread_local std::string g_last_error;

edit_status_t fail(edit_status_t s, const std::string& msg) {
  g_last_error = msg;
  return s;
}

edit_status_t fail_hip(hipError_t e, const char* what) {
  return fail(EDIT_EHIP, std::string(what) + ": " + hipGetErrorString(e));
}

struct Unit {
  int64_t n = 0;
  int rows = 1;         // pass-1 blocks = partial rows (one-pass mode: fused blocks)
  int blocks2 = 1;      // pass-2 blocks
  double* partials = nullptr;
  UnitRecord* rec = nullptr;
  hipEvent_t done = nullptr;
  hipEvent_t prof[4] = {nullptr, nullptr, nullptr, nullptr};
  bool pending = false;   // a completion to wait for has been recorded
  int done_slot = -1;     // -1: `done` (a single step); else the round-event slot
  uint64_t done_gen = 0;  // generation of that slot's record the unit belongs to
  bool profiled = false;  // prof[] hold the last step's timestamps
  bool has_state = false; // stepped or state_set at least once
};

}  // namespace

namespace {

// Staging of theta and momentum for rounds whose master copies live in host
// memory: a ring of device slots, one stream per copy direction, and per
// slot the events that order copy-in -> compute -> copy-out -> reuse.
constexpr int kOffloadSlots = 3;

struct Offload {
  int64_t cap = 0;           // elements per slot (theta and b each)
  float* buf = nullptr;      // [kOffloadSlots][2][cap] fp32
  hipStream_t h2d = nullptr, d2h = nullptr;
  hipEvent_t in_done[kOffloadSlots] = {};
  hipEvent_t comp_done[kOffloadSlots] = {};
  hipEvent_t out_done[kOffloadSlots] = {};
  hipEvent_t start = nullptr;  // the caller's stream at the start of a round
  bool used[kOffloadSlots] = {};
  bool ready = false;
};

}  // namespace

// Device scratch of edit_outer_step_layer_noalloc: the per-block Gram partials
// of one step, in a fixed array that each GPU holds for the life of the
// process (no allocation per call).  Host code never names the array itself
// (on the host `scratch` is only a stand-in for the symbol): its device
// address comes from hipGetSymbolAddress, taken once per device at the first
// edit_outer_init on that device, with that device current.
constexpr size_t kNoAllocScratchBytes = size_t(1) << 20;  // EDIT_NOALLOC_SCRATCH_BYTES
static_assert(kNoAllocScratchBytes == EDIT_NOALLOC_SCRATCH_BYTES, "header and library disagree");
static __device__ __align__(256) double scratch[kNoAllocScratchBytes / sizeof(double)];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mutex;
void* g_scratch_ptr[kMaxDevices] = {};  // device address of `scratch` on each device

// The device address of the scratch array on `device` (current), looked up
// on first use.
edit_status_t noalloc_scratch(int device, void** out) {
  if (device < 0 || device >= kMaxDevices)
    return fail(EDIT_EINVAL, "device index " + std::to_string(device) + " beyond the scratch table");
  std::lock_guard<std::mutex> lock(g_scratch_mutex);
  if (!g_scratch_ptr[device]) {
    void* ptr = nullptr;
    const hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !ptr) return fail_hip(e, "hipGetSymbolAddress(scratch)");
    g_scratch_ptr[device] = ptr;
  }
  *out = g_scratch_ptr[device];
  return EDIT_OK;
}

}  // namespace

struct edit_outer {
  edit_outer_config_t cfg{};
  std::vector<int64_t> numel;
  int device = 0;
  int num_cu = 0;
  int pass2_lds = 0;       // dynamic LDS per update-pass block (occupancy cap)
  int fused_lds = 0;       // the same for the one-pass kernel
  int cap1 = 1;            // resident blocks of pass 1 on the whole GPU
  int32_t profile_every = 0;  // record kernel events on units l with l % every == 0
  char* arena = nullptr;   // one device allocation for every unit's scratch
  void* noalloc = nullptr; // this device's fixed scratch array (step_layer_noalloc)
  FinishEntry* finish_table = nullptr;  // one-pass mode: [L] entries, in the arena
  bool one_pass = false;
  Offload off;
  std::vector<Unit> units;
  // Completion of a round: one event recorded after its last kernel, shared
  // by its units (an event record costs a few microseconds of stream time,
  // one per unit would cost ~1% of a 1B round).  A ring of slots; before a
  // slot is recorded again the host waits for its previous record, so every
  // generation up to round_complete[slot] is known to have finished.
  static constexpr int kRoundEvents = 4;
  hipEvent_t round_ev[kRoundEvents] = {};
  uint64_t round_gen[kRoundEvents] = {};       // generation of the slot's latest record
  uint64_t round_complete[kRoundEvents] = {};  // generations <= this have finished
  uint64_t next_gen = 1;
  int next_slot = 0;
};

namespace {

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

edit_status_t check_device(const edit_outer* h) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail_hip(e, "hipGetDevice");
  if (dev != h->device)
    return fail(EDIT_EINVAL, "call made with device " + std::to_string(dev) +
                                 " current; the handle belongs to device " +
                                 std::to_string(h->device));
  return EDIT_OK;
}

void destroy_offload(edit_outer* h) {
  Offload& o = h->off;
  if (o.h2d) (void)hipStreamSynchronize(o.h2d);
  if (o.d2h) (void)hipStreamSynchronize(o.d2h);
  for (int s = 0; s < kOffloadSlots; ++s) {
    if (o.in_done[s]) (void)hipEventDestroy(o.in_done[s]);
    if (o.comp_done[s]) (void)hipEventDestroy(o.comp_done[s]);
    if (o.out_done[s]) (void)hipEventDestroy(o.out_done[s]);
  }
  if (o.start) (void)hipEventDestroy(o.start);
  if (o.h2d) (void)hipStreamDestroy(o.h2d);
  if (o.d2h) (void)hipStreamDestroy(o.d2h);
  if (o.buf) (void)hipFree(o.buf);
  o = Offload{};
}

void destroy_units(edit_outer* h) {
  destroy_offload(h);
  for (hipEvent_t& ev : h->round_ev)
    if (ev) {
      (void)hipEventDestroy(ev);
      ev = nullptr;
    }
  for (Unit& u : h->units) {
    if (u.done) (void)hipEventDestroy(u.done);
    for (hipEvent_t& ev : u.prof)
      if (ev) (void)hipEventDestroy(ev);
  }
  h->units.clear();
  if (h->arena) (void)hipFree(h->arena);
  h->arena = nullptr;
}

}  // namespace

namespace edit {

edit_status_t set_error(edit_status_t s, const char* msg) { return fail(s, msg); }

edit_status_t validate_config(const edit_outer_config_t* cfg) {
  const int K = cfg->num_workers;
  if (K < 1 || K > EDIT_MAX_K)
    return fail(EDIT_EINVAL, "num_workers must be in 1.." + std::to_string(EDIT_MAX_K));
  if (cfg->num_layers < 1) return fail(EDIT_EINVAL, "num_layers must be >= 1");
  if (!cfg->layer_numel) return fail(EDIT_EINVAL, "layer_numel must not be NULL");
  if (cfg->replica_dtype != EDIT_F32 && cfg->replica_dtype != EDIT_BF16)
    return fail(EDIT_EINVAL, "replica_dtype must be EDIT_F32 or EDIT_BF16");
  if (cfg->flags & ~(EDIT_AE | EDIT_WA | EDIT_GC | EDIT_ONE_PASS))
    return fail(EDIT_EINVAL, "unknown flag bits");
  if ((cfg->flags & EDIT_ONE_PASS) && (cfg->flags & (EDIT_AE | EDIT_WA | EDIT_GC)))
    return fail(EDIT_EINVAL, "flag EDIT_ONE_PASS needs EDIT_AE, EDIT_WA and EDIT_GC clear");
  if (!(cfg->ema_alpha > 0.0 && cfg->ema_alpha <= 1.0))
    return fail(EDIT_EINVAL, "ema_alpha must be in (0, 1]");
  if (!(cfg->clip_eps > 0.0)) return fail(EDIT_EINVAL, "clip_eps must be > 0");
  if (!(cfg->clip_threshold >= 0.0)) return fail(EDIT_EINVAL, "clip_threshold must be >= 0");
  if (!std::isfinite(cfg->outer_lr) || !std::isfinite(cfg->momentum) ||
      !std::isfinite(cfg->z_threshold))
    return fail(EDIT_EINVAL, "outer_lr, momentum and z_threshold must be finite");
  if (cfg->ema_warmup_rounds < 0) return fail(EDIT_EINVAL, "ema_warmup_rounds must be >= 0");
  if (cfg->flags & EDIT_AE) {
    const int64_t w_min = edit_outer_min_warmup(cfg->ema_alpha, cfg->z_threshold);
    if (w_min < 0)
      return fail(EDIT_EINVAL, "z_threshold must be > 0 with EDIT_AE: no EMA warm-up lets a worker "
                               "with a steady norm pass the z-test");
    if (cfg->ema_warmup_rounds < w_min) {
      char msg[200];
      std::snprintf(msg, sizeof msg,
                    "ema_warmup_rounds must be >= %lld for ema_alpha = %g and z_threshold = %g: a "
                    "shorter warm-up flags every worker with a steady norm for good",
                    static_cast<long long>(w_min), cfg->ema_alpha, cfg->z_threshold);
      return fail(EDIT_EINVAL, msg);
    }
  }
  for (int l = 0; l < cfg->num_layers; ++l)
    if (cfg->layer_numel[l] < 0)
      return fail(EDIT_EINVAL, "layer_numel[" + std::to_string(l) + "] is negative");
  return EDIT_OK;
}

edit_status_t current_gfx950(int* device, int* num_cu) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail_hip(e, "hipGetDevice");
  hipDeviceProp_t prop;
  e = hipGetDeviceProperties(&prop, dev);
  if (e != hipSuccess) return fail_hip(e, "hipGetDeviceProperties");
  if (std::strncmp(prop.gcnArchName, "gfx950", 6) != 0)
    return fail(EDIT_ENODEV, std::string("device arch is ") + prop.gcnArchName +
                                 "; this library is built for gfx950 only");
  *device = dev;
  *num_cu = prop.multiProcessorCount;
  return EDIT_OK;
}

}  // namespace edit

extern "C" {

// The z-test of Eq. 1 against the EMA state after k updates by a norm that
// stays G every round, from the zero state: mu_k = G(1 - (1-alpha)^k) lags
// G, so a clean worker passes only once k is large enough.  The recurrence
// is homogeneous in G, so G = 1 stands for every G > 0.
int64_t edit_outer_min_warmup(double alpha, double delta) {
  if (!(alpha > 0.0 && alpha <= 1.0) || !std::isfinite(delta)) return -1;
  constexpr int64_t kSearch = 1 << 20;  // z falls like (1-alpha)^(k/2): far beyond any alpha in use
  const double G = 1.0;
  double mu = 0.0, sigma = 0.0;
  for (int64_t k = 0; k <= kSearch; ++k) {
    if (!((G - mu) > delta * sigma)) return k;
    const double m = alpha * G + (1.0 - alpha) * mu;
    const double dev = G - m;
    sigma = std::sqrt((1.0 - alpha) * sigma * sigma + alpha * dev * dev);
    mu = m;
  }
  return -1;
}

const char* edit_outer_strerror(edit_status_t s) {
  switch (s) {
    case EDIT_OK: return "ok";
    case EDIT_EINVAL: return "invalid argument";
    case EDIT_ENOMEM: return "out of memory";
    case EDIT_EHIP: return "HIP runtime error";
    case EDIT_ESTATE: return "invalid state";
    case EDIT_ENODEV: return "no gfx950 device";
  }
  return "unknown status";
}

const char* edit_outer_last_error(void) { return g_last_error.c_str(); }

edit_status_t edit_outer_init(const edit_outer_config_t* cfg, edit_outer_t* out) {
  g_last_error.clear();
  if (!cfg || !out) return fail(EDIT_EINVAL, "cfg and out must not be NULL");
  *out = nullptr;
  const int K = cfg->num_workers;
  EDIT_TRY(validate_config(cfg));
  int dev = 0, num_cu = 0;
  EDIT_TRY(current_gfx950(&dev, &num_cu));
  void* noalloc = nullptr;
  EDIT_TRY(noalloc_scratch(dev, &noalloc));
  hipError_t e = hipSuccess;

  edit_outer* h = new (std::nothrow) edit_outer;
  if (!h) return fail(EDIT_ENOMEM, "host allocation failed");
  h->cfg = *cfg;
  h->numel.assign(cfg->layer_numel, cfg->layer_numel + cfg->num_layers);
  h->cfg.layer_numel = h->numel.data();
  h->device = dev;
  h->num_cu = num_cu;
  {
    int lds_per_cu = 0;
    e = hipDeviceGetAttribute(&lds_per_cu, hipDeviceAttributeMaxSharedMemoryPerMultiprocessor, dev);
    if (e != hipSuccess) {
      delete h;
      return fail_hip(e, "hipDeviceGetAttribute(LDS per CU)");
    }
    h->pass2_lds = update_pass_lds(K, lds_per_cu);
    h->fused_lds = one_pass_lds(K, cfg->replica_dtype == EDIT_BF16, lds_per_cu);
  }
  h->noalloc = noalloc;
  const bool bf16 = cfg->replica_dtype == EDIT_BF16;
  h->cap1 = h->num_cu * pass1_blocks_per_cu(K, bf16);
  h->one_pass = (cfg->flags & EDIT_ONE_PASS) != 0;

  // Lay out every unit's record and partials in one allocation.
  const int ve = bf16 ? 8 : 4;
  const size_t rec_bytes = (sizeof(UnitRecord) + 255) & ~size_t(255);
  size_t total = 0;
  h->units.resize(cfg->num_layers);
  std::vector<size_t> offs(cfg->num_layers);
  for (int l = 0; l < cfg->num_layers; ++l) {
    Unit& u = h->units[l];
    u.n = h->numel[l];
    const int64_t nvec = u.n / ve;
    // one resident slot stays free for the block that takes the previous
    // unit's decision in a round (and step_layer uses the same rows, so both
    // paths reduce in the same order)
    u.rows = static_cast<int>(
        std::max<int64_t>(1, std::min<int64_t>(h->cap1 - 1, ceil_div(nvec, kThreads))));
    // pass 2 (and the one-pass kernel): a fixed number of vectors per thread,
    // so the block count grows with the unit
    if (ceil_div(nvec, kPass2Threads) > INT32_MAX) {
      delete h;
      return fail(EDIT_EINVAL, "layer_numel[" + std::to_string(l) + "] is too large");
    }
    u.blocks2 = static_cast<int>(std::max<int64_t>(1, ceil_div(nvec, kPass2Threads)));
    if (h->one_pass)
      u.rows = static_cast<int>(std::max<int64_t>(
          1, ceil_div(nvec, int64_t(kFusedThreads) * fused_vectors_per_thread(K, bf16))));
    offs[l] = total;
    const size_t per_row = h->one_pass ? size_t(K + 1) : size_t(num_pairs(K));
    const size_t part_bytes = (per_row * u.rows * sizeof(double) + 255) & ~size_t(255);
    total += rec_bytes + part_bytes;
  }
  const size_t table_off = total;
  if (h->one_pass) total += (sizeof(FinishEntry) * cfg->num_layers + 255) & ~size_t(255);
  e = hipMalloc(reinterpret_cast<void**>(&h->arena), total);
  if (e != hipSuccess) {
    delete h;
    return fail(EDIT_ENOMEM, std::string("hipMalloc of scratch: ") + hipGetErrorString(e));
  }
  e = hipMemset(h->arena, 0, total);  // EMA state mu = sigma = 0, round 0
  for (int l = 0; l < cfg->num_layers && e == hipSuccess; ++l) {
    Unit& u = h->units[l];
    u.rec = reinterpret_cast<UnitRecord*>(h->arena + offs[l]);
    u.partials = reinterpret_cast<double*>(h->arena + offs[l] + rec_bytes);
    e = hipEventCreateWithFlags(&u.done, hipEventDisableTiming);
  }
  if (e == hipSuccess && h->one_pass) {
    std::vector<FinishEntry> table(cfg->num_layers);
    for (int l = 0; l < cfg->num_layers; ++l)
      table[l] = {h->units[l].partials, h->units[l].rec, h->units[l].rows, 0};
    h->finish_table = reinterpret_cast<FinishEntry*>(h->arena + table_off);
    e = hipMemcpy(h->finish_table, table.data(), sizeof(FinishEntry) * table.size(),
                  hipMemcpyHostToDevice);
  }
  if (e == hipSuccess) e = hipDeviceSynchronize();
  if (e != hipSuccess) {
    destroy_units(h);
    delete h;
    return fail_hip(e, "init");
  }
  *out = h;
  return EDIT_OK;
}

}  // extern "C"

namespace {

// Argument checks shared by the step entry points.  `momentum` may be NULL
// only when `need_momentum` is false (the Gram pass does not touch it).
// `extra`, when not NULL, is one more buffer of `extra_bytes` (a Gram vector)
// that must not overlap the others.
edit_status_t check_step(const edit_outer* h, int32_t layer, const float* theta,
                         const float* momentum, void* const* replicas,
                         bool need_momentum = true, const void* extra = nullptr,
                         int64_t extra_bytes = 0) {
  if (layer < 0 || layer >= h->cfg.num_layers)
    return fail(EDIT_EINVAL, "layer " + std::to_string(layer) + " out of range");
  const Unit& u = h->units[layer];
  const int K = h->cfg.num_workers;
  const int64_t n = u.n;
  if (n == 0) return EDIT_OK;
  if (!replicas) return fail(EDIT_EINVAL, "replicas must not be NULL");
  if (!theta || (need_momentum && !momentum))
    return fail(EDIT_EINVAL, "theta and momentum must not be NULL");
  if (!aligned16(theta) || (momentum && !aligned16(momentum)))
    return fail(EDIT_EINVAL, "theta and momentum must be 16-byte aligned");
  // Every buffer's byte range, for the alias check.
  struct Range {
    uintptr_t lo, hi;
  };
  Range r[EDIT_MAX_K + 3];
  int nr = 0;
  r[nr++] = {reinterpret_cast<uintptr_t>(theta), reinterpret_cast<uintptr_t>(theta) + 4 * n};
  if (momentum)
    r[nr++] = {reinterpret_cast<uintptr_t>(momentum), reinterpret_cast<uintptr_t>(momentum) + 4 * n};
  if (extra)
    r[nr++] = {reinterpret_cast<uintptr_t>(extra), reinterpret_cast<uintptr_t>(extra) + extra_bytes};
  const int64_t rb = h->cfg.replica_dtype == EDIT_BF16 ? 2 : 4;
  for (int j = 0; j < K; ++j) {
    if (!replicas[j]) return fail(EDIT_EINVAL, "replica pointer " + std::to_string(j) + " is NULL");
    if (!aligned16(replicas[j]))
      return fail(EDIT_EINVAL, "replica " + std::to_string(j) + " is not 16-byte aligned");
    const uintptr_t p = reinterpret_cast<uintptr_t>(replicas[j]);
    r[nr++] = {p, p + rb * n};
  }
  for (int a = 0; a < nr; ++a)
    for (int b = a + 1; b < nr; ++b)
      if (r[a].lo < r[b].hi && r[b].lo < r[a].hi)
        return fail(EDIT_EINVAL, extra ? "theta, momentum, the replicas and gram must not overlap"
                                       : "theta, momentum and the replicas must not overlap");
  return EDIT_OK;
}

// A Gram vector argument: non-NULL and 8-byte aligned.
edit_status_t check_gram(const void* gram) {
  if (!gram) return fail(EDIT_EINVAL, "gram must not be NULL");
  if (reinterpret_cast<uintptr_t>(gram) & 7u) return fail(EDIT_EINVAL, "gram must be 8-byte aligned");
  return EDIT_OK;
}

DecideParams decide_params(const edit_outer* h) {
  DecideParams prm;
  prm.alpha = h->cfg.ema_alpha;
  prm.delta = h->cfg.z_threshold;
  prm.phi = h->cfg.clip_threshold;
  prm.eps = h->cfg.clip_eps;
  prm.warmup = h->cfg.ema_warmup_rounds;
  prm.flags = h->cfg.flags;
  return prm;
}

static void* const kNoReplicas[EDIT_MAX_K] = {};

// Enqueue helpers; each returns EDIT_OK or the failure (message already set).
struct Enqueue {
  edit_outer* h;
  hipStream_t s;
  DecideParams prm;
  int K;
  bool bf16;

  bool profiled(int32_t layer) const {
    return h->profile_every > 0 && layer % h->profile_every == 0;
  }
  edit_status_t event(Unit& u, int32_t layer, int k) {
    if (!profiled(layer)) return EDIT_OK;
    hipError_t e = hipSuccess;
    // timing only: no system-scope fence (it would add stream time)
    if (!u.prof[k] && (e = hipEventCreateWithFlags(&u.prof[k], hipEventDisableSystemFence)) != hipSuccess)
      return fail_hip(e, "hipEventCreate");
    if ((e = hipEventRecord(u.prof[k], s)) != hipSuccess) return fail_hip(e, "hipEventRecord");
    return EDIT_OK;
  }
  // pass 1 of `layer`, optionally with the decision of `prev` in the same launch
  edit_status_t pass1(int32_t layer, const float* theta, void* const* replicas, Unit* prev) {
    Unit& u = h->units[layer];
    const void* const* creps =
        u.n == 0 ? kNoReplicas : const_cast<const void* const*>(replicas);
    hipError_t e = launch_pass1(K, bf16, u.rows, theta, creps, u.n, u.partials,
                                prev ? prev->partials : nullptr, prev ? prev->rows : 0,
                                prev ? prev->rec : nullptr, prm, s);
    return e == hipSuccess ? EDIT_OK : fail_hip(e, "pass1 launch");
  }
  // pass 1 of one or two units (K <= 8) in one launch, whose block 0 takes
  // the decisions of `nprev` earlier units first
  edit_status_t pass1_pair(const int32_t* layer, float* const* theta, void* const* const* replicas,
                           int count, const int32_t* prev, int nprev) {
    Pass1Desc unit[2];
    for (int i = 0; i < count; ++i) {
      const Unit& u = h->units[layer[i]];
      unit[i] = {theta[i], u.n == 0 ? kNoReplicas : const_cast<const void* const*>(replicas[i]), u.n,
                 u.partials, u.rows};
    }
    DecideDesc dd[2];
    describe(prev, nprev, dd);
    hipError_t e = launch_pass1_pair(K, bf16, unit, count, dd, nprev, prm, s);
    return e == hipSuccess ? EDIT_OK : fail_hip(e, "pass1 launch");
  }
  // a small launch: the decisions of `nprev` earlier units and whole
  // single-block units
  edit_status_t small(const int32_t* prev, int nprev, const SingleBlockDesc* single, int nsingle) {
    DecideDesc dd[2];
    describe(prev, nprev, dd);
    hipError_t e = launch_round_small(K, bf16, dd, nprev, prm, single, nsingle, h->cfg.outer_lr,
                                      h->cfg.momentum, s);
    return e == hipSuccess ? EDIT_OK : fail_hip(e, "small launch");
  }
  void describe(const int32_t* layer, int count, DecideDesc* dd) const {
    for (int i = 0; i < count; ++i) {
      const Unit& u = h->units[layer[i]];
      dd[i] = {u.partials, u.rows, u.rec};
    }
  }
  edit_status_t gram_out(int32_t layer, double* gram) {
    Unit& u = h->units[layer];
    hipError_t e = launch_gram_reduce(K, u.partials, u.rows, gram, s);
    return e == hipSuccess ? EDIT_OK : fail_hip(e, "gram reduce launch");
  }
  edit_status_t decide_from(int32_t layer, const double* gram) {
    Unit& u = h->units[layer];
    hipError_t e = launch_decide_gram(K, gram, u.rec, prm, s);
    return e == hipSuccess ? EDIT_OK : fail_hip(e, "decide launch");
  }
  edit_status_t decide(int32_t layer) {
    Unit& u = h->units[layer];
    hipError_t e = launch_decide(K, u.partials, u.rows, u.rec, prm, s);
    return e == hipSuccess ? EDIT_OK : fail_hip(e, "decide launch");
  }
  edit_status_t pass2(int32_t layer, float* theta, float* momentum, void* const* replicas) {
    Unit& u = h->units[layer];
    void* const* mreps = u.n == 0 ? kNoReplicas : replicas;
    hipError_t e = launch_pass2(K, bf16, u.blocks2, h->pass2_lds, theta, momentum, mreps, u.rec, u.n,
                                h->cfg.outer_lr, h->cfg.momentum, s);
    if (e != hipSuccess) return fail_hip(e, "pass2 launch");
    return EDIT_OK;
  }
  // one-pass mode: the fused pass of `layer`, and the record reduction of
  // `units` table entries from `first` (marked units only)
  edit_status_t fused(int32_t layer, float* theta, float* momentum, void* const* replicas) {
    Unit& u = h->units[layer];
    void* const* mreps = u.n == 0 ? kNoReplicas : replicas;
    hipError_t e = launch_fused_mean(K, bf16, u.rows, h->fused_lds, theta, momentum, mreps, u.partials, u.rec, u.n,
                                     h->cfg.outer_lr, h->cfg.momentum, s);
    return e == hipSuccess ? EDIT_OK : fail_hip(e, "one-pass launch");
  }
  edit_status_t records(int32_t first, int32_t units) {
    hipError_t e = launch_fused_finish(K, h->finish_table + first, units, s);
    return e == hipSuccess ? EDIT_OK : fail_hip(e, "record launch");
  }
  edit_status_t finish(int32_t layer) {
    Unit& u = h->units[layer];
    hipError_t e = hipEventRecord(u.done, s);
    if (e != hipSuccess) return fail_hip(e, "hipEventRecord");
    u.pending = true;
    u.done_slot = -1;
    u.profiled = profiled(layer);
    u.has_state = true;
    return EDIT_OK;
  }
  // The end of a round: one event for all of its units.
  edit_status_t finish_round(const int32_t* layers, int32_t count) {
    const int slot = h->next_slot;
    h->next_slot = (slot + 1) % edit_outer::kRoundEvents;
    hipError_t e = hipSuccess;
    if (!h->round_ev[slot] && (e = hipEventCreateWithFlags(&h->round_ev[slot], hipEventDisableTiming)) != hipSuccess)
      return fail_hip(e, "hipEventCreate");
    if (h->round_gen[slot] > h->round_complete[slot]) {  // its previous round may still run
      if ((e = hipEventSynchronize(h->round_ev[slot])) != hipSuccess) return fail_hip(e, "hipEventSynchronize");
      h->round_complete[slot] = h->round_gen[slot];
    }
    if ((e = hipEventRecord(h->round_ev[slot], s)) != hipSuccess) return fail_hip(e, "hipEventRecord");
    const uint64_t gen = h->next_gen++;
    h->round_gen[slot] = gen;
    for (int32_t i = 0; i < count; ++i) {
      Unit& u = h->units[layers[i]];
      u.pending = true;
      u.done_slot = slot;
      u.done_gen = gen;
      u.profiled = profiled(layers[i]);
      u.has_state = true;
    }
    return EDIT_OK;
  }
};

// Wait until the last enqueued step of `u` has finished.
edit_status_t wait_unit(edit_outer* h, Unit& u) {
  if (!u.pending) return EDIT_OK;
  hipError_t e = hipSuccess;
  if (u.done_slot < 0) {
    e = hipEventSynchronize(u.done);
  } else {
    const int slot = u.done_slot;
    if (h->round_complete[slot] >= u.done_gen) return EDIT_OK;
    // not recorded again since (that would have completed this generation)
    e = hipEventSynchronize(h->round_ev[slot]);
    if (e == hipSuccess) h->round_complete[slot] = h->round_gen[slot];
  }
  return e == hipSuccess ? EDIT_OK : fail_hip(e, "hipEventSynchronize");
}


}  // namespace

extern "C" {

edit_status_t edit_outer_step_layer(edit_outer_t h, int32_t layer, float* theta, float* momentum,
                                    void* const* replicas, void* stream) {
  if (!h) return fail(EDIT_EINVAL, "NULL handle");
  EDIT_TRY(check_step(h, layer, theta, momentum, replicas));
  EDIT_TRY(check_device(h));
  Enqueue q{h, reinterpret_cast<hipStream_t>(stream), decide_params(h), h->cfg.num_workers,
            h->cfg.replica_dtype == EDIT_BF16};
  if (h->one_pass) {
    EDIT_TRY(q.event(h->units[layer], layer, 0));
    EDIT_TRY(q.fused(layer, theta, momentum, replicas));
    EDIT_TRY(q.event(h->units[layer], layer, 1));
    EDIT_TRY(q.event(h->units[layer], layer, 2));
    EDIT_TRY(q.records(layer, 1));
    EDIT_TRY(q.event(h->units[layer], layer, 3));
    return q.finish(layer);
  }
  EDIT_TRY(q.event(h->units[layer], layer, 0));
  EDIT_TRY(q.pass1(layer, theta, replicas, nullptr));
  EDIT_TRY(q.decide(layer));
  EDIT_TRY(q.event(h->units[layer], layer, 1));
  EDIT_TRY(q.event(h->units[layer], layer, 2));
  EDIT_TRY(q.pass2(layer, theta, momentum, replicas));
  EDIT_TRY(q.event(h->units[layer], layer, 3));
  return q.finish(layer);
}

edit_status_t edit_outer_step_layer_noalloc(edit_outer_t h, int32_t layer, float* theta, float* momentum,
                                            void* const* replicas, void* stream) {
  if (!h) return fail(EDIT_EINVAL, "NULL handle");
  if (h->one_pass) return fail(EDIT_EINVAL, "edit_outer_step_layer_noalloc is not available with EDIT_ONE_PASS");
  EDIT_TRY(check_step(h, layer, theta, momentum, replicas));
  const int K = h->cfg.num_workers;
  Unit& u = h->units[layer];
  const size_t need = static_cast<size_t>(num_pairs(K)) * static_cast<size_t>(u.rows) * sizeof(double);
  if (need > kNoAllocScratchBytes)
    return fail(EDIT_EINVAL, "unit " + std::to_string(layer) + " needs " + std::to_string(need) +
                                 " bytes of partial sums; the fixed scratch holds " +
                                 std::to_string(kNoAllocScratchBytes));
  EDIT_TRY(check_device(h));
  const hipStream_t s = reinterpret_cast<hipStream_t>(stream);
  const bool bf16 = h->cfg.replica_dtype == EDIT_BF16;
  const DecideParams prm = decide_params(h);
  double* partials = static_cast<double*>(h->noalloc);  // the device address, never `scratch` itself
  const void* const* creps = u.n == 0 ? kNoReplicas : const_cast<const void* const*>(replicas);
  hipError_t e = launch_pass1(K, bf16, u.rows, theta, creps, u.n, partials, nullptr, 0, nullptr, prm, s);
  if (e != hipSuccess) return fail_hip(e, "pass1 launch");
  if ((e = launch_decide(K, partials, u.rows, u.rec, prm, s)) != hipSuccess) return fail_hip(e, "decide launch");
  Enqueue q{h, s, prm, K, bf16};
  EDIT_TRY(q.pass2(layer, theta, momentum, replicas));
  if ((e = hipEventRecord(u.done, s)) != hipSuccess) return fail_hip(e, "hipEventRecord");
  u.pending = true;
  u.done_slot = -1;
  u.profiled = false;
  u.has_state = true;
  return EDIT_OK;
}

edit_status_t edit_outer_gram_layer(edit_outer_t h, int32_t layer, const float* theta,
                                    void* const* replicas, double* gram, void* stream) {
  if (!h) return fail(EDIT_EINVAL, "NULL handle");
  if (h->one_pass) return fail(EDIT_EINVAL, "the Gram entry points are not available with EDIT_ONE_PASS");
  EDIT_TRY(check_gram(gram));
  const int K = h->cfg.num_workers;
  EDIT_TRY(check_step(h, layer, theta, nullptr, replicas, false, gram,
                      static_cast<int64_t>(num_pairs(K)) * 8));
  EDIT_TRY(check_device(h));
  Enqueue q{h, reinterpret_cast<hipStream_t>(stream), decide_params(h), K,
            h->cfg.replica_dtype == EDIT_BF16};
  EDIT_TRY(q.pass1(layer, theta, replicas, nullptr));
  return q.gram_out(layer, gram);
}

edit_status_t edit_outer_apply_layer(edit_outer_t h, int32_t layer, const double* gram,
                                     float* theta, float* momentum, void* const* replicas,
                                     void* stream) {
  if (!h) return fail(EDIT_EINVAL, "NULL handle");
  if (h->one_pass) return fail(EDIT_EINVAL, "the Gram entry points are not available with EDIT_ONE_PASS");
  EDIT_TRY(check_gram(gram));
  const int K = h->cfg.num_workers;
  EDIT_TRY(check_step(h, layer, theta, momentum, replicas, true, gram,
                      static_cast<int64_t>(num_pairs(K)) * 8));
  EDIT_TRY(check_device(h));
  Enqueue q{h, reinterpret_cast<hipStream_t>(stream), decide_params(h), K,
            h->cfg.replica_dtype == EDIT_BF16};
  Unit& u = h->units[layer];
  EDIT_TRY(q.event(u, layer, 0));
  EDIT_TRY(q.decide_from(layer, gram));
  EDIT_TRY(q.event(u, layer, 1));
  EDIT_TRY(q.event(u, layer, 2));
  EDIT_TRY(q.pass2(layer, theta, momentum, replicas));
  EDIT_TRY(q.event(u, layer, 3));
  return q.finish(layer);
}

edit_status_t edit_outer_step_round(edit_outer_t h, int32_t count, const int32_t* layers,
                                    float* const* theta, float* const* momentum,
                                    void* const* replicas, void* stream) {
  if (!h) return fail(EDIT_EINVAL, "NULL handle");
  if (count < 1) return fail(EDIT_EINVAL, "count must be >= 1");
  if (!layers || !theta || !momentum || !replicas)
    return fail(EDIT_EINVAL, "layers, theta, momentum and replicas must not be NULL");
  const int K = h->cfg.num_workers;
  std::vector<char> seen(h->cfg.num_layers, 0);
  for (int32_t i = 0; i < count; ++i) {
    EDIT_TRY(check_step(h, layers[i], theta[i], momentum[i], replicas + static_cast<size_t>(i) * K));
    if (seen[layers[i]]++)
      return fail(EDIT_EINVAL, "layer " + std::to_string(layers[i]) + " appears twice in a round");
  }
  EDIT_TRY(check_device(h));
  Enqueue q{h, reinterpret_cast<hipStream_t>(stream), decide_params(h), K,
            h->cfg.replica_dtype == EDIT_BF16};
  if (h->one_pass) {
    // No later kernel of the round needs a unit's record, so the fused passes
    // run back to back and one launch then reduces every stepped unit's norms.
    for (int32_t i = 0; i < count; ++i) {
      const int32_t l = layers[i];
      EDIT_TRY(q.event(h->units[l], l, 0));
      EDIT_TRY(q.fused(l, theta[i], momentum[i], replicas + static_cast<size_t>(i) * K));
      EDIT_TRY(q.event(h->units[l], l, 1));
      EDIT_TRY(q.event(h->units[l], l, 2));
      EDIT_TRY(q.event(h->units[l], l, 3));
    }
    EDIT_TRY(q.records(0, h->cfg.num_layers));
    return q.finish_round(layers, count);
  }
  // Up to K = 8 every unit's decision rides in the next pass-1 launch
  // (one extra block, which would otherwise idle), and its pass 2 follows
  // that launch; the one-block decision then never holds up the whole chip
  // (measured at the 1B shape, same box: 14.63-14.68 ms per round against
  // 14.79 ms with a decision kernel between each unit's two passes).  Two
  // consecutive units also share one pass-1 launch (not the round's last
  // unit, whose decision would then wait for the other's), so the persistent
  // grid starts and drains once per pair; the next launch then takes both
  // decisions.  Above K = 8 the Gram pass is bound by fp64 arithmetic and
  // reads through the cache, so a unit's pass 2 instead follows its own pass
  // 1 with only the decision between them and finds the end of its input in
  // the Infinity Cache (measured at K = 16: 696 against 730 us per
  // 51.4M-element pass 2).
  //
  // A unit whose Gram pass is one block is stepped whole by one block of a
  // small launch, up to kMaxSingleBlockUnits per launch (its own two
  // launches cost about 16 us at K = 16, its work a few microseconds); a
  // small launch also carries the pending decisions.  Such units are
  // independent of the others, so this only changes which launch runs them.
  // Units whose kernels are being timed keep their own launches.
  const bool adjacent = K > 8;
  int32_t pend[2];  // indices i of the units whose decisions are not launched yet
  int32_t pend_layer[2];
  int npend = 0;
  SingleBlockDesc single[kMaxSingleBlockUnits];
  int nsingle = 0;
  auto reps_of = [&](int32_t i) { return replicas + static_cast<size_t>(i) * K; };
  auto rider = [&](int32_t i) { return h->units[layers[i]].rows == 1 && !q.profiled(layers[i]); };
  // pass 2 of the pending units, whose decisions the last launch took
  auto flush_pass2 = [&]() -> edit_status_t {
    for (int k = 0; k < npend; ++k) {
      const int32_t i = pend[k], l = layers[i];
      EDIT_TRY(q.event(h->units[l], l, 2));
      EDIT_TRY(q.pass2(l, theta[i], momentum[i], reps_of(i)));
      EDIT_TRY(q.event(h->units[l], l, 3));
    }
    npend = 0;
    return EDIT_OK;
  };
  // the pending decisions and the waiting single-block units, then the
  // pending units' pass 2
  auto flush_small = [&]() -> edit_status_t {
    EDIT_TRY(q.small(pend_layer, npend, single, nsingle));
    nsingle = 0;
    return flush_pass2();
  };
  for (int32_t i = 0; i < count; ++i) {
    const int32_t l = layers[i];
    Unit& u = h->units[l];
    if (rider(i)) {
      single[nsingle++] = {theta[i], momentum[i], reps_of(i), u.partials, u.rec, u.n};
      if (nsingle == kMaxSingleBlockUnits) EDIT_TRY(flush_small());
      continue;
    }
    if (nsingle > 0) {
      EDIT_TRY(flush_small());
    } else if (adjacent && npend > 0) {
      EDIT_TRY(q.decide(pend_layer[0]));
      EDIT_TRY(flush_pass2());
    }
    const bool pair = !adjacent && !q.profiled(l) && i + 2 < count && !rider(i + 1) &&
                      !q.profiled(layers[i + 1]);
    if (pair) {
      float* const th2[2] = {theta[i], theta[i + 1]};
      void* const* const rp2[2] = {reps_of(i), reps_of(i + 1)};
      EDIT_TRY(q.pass1_pair(layers + i, th2, rp2, 2, pend_layer, npend));
      EDIT_TRY(flush_pass2());
      pend[0] = i, pend_layer[0] = l;
      pend[1] = i + 1, pend_layer[1] = layers[i + 1];
      npend = 2;
      ++i;
      continue;
    }
    EDIT_TRY(q.event(u, l, 0));
    if (npend == 2) {  // both decisions of the pair before it
      float* const th1[1] = {theta[i]};
      void* const* const rp1[1] = {reps_of(i)};
      EDIT_TRY(q.pass1_pair(layers + i, th1, rp1, 1, pend_layer, npend));
    } else {
      EDIT_TRY(q.pass1(l, theta[i], reps_of(i), npend ? &h->units[pend_layer[0]] : nullptr));
    }
    EDIT_TRY(q.event(u, l, 1));
    EDIT_TRY(flush_pass2());
    pend[0] = i, pend_layer[0] = l;
    npend = 1;
  }
  if (nsingle > 0 || npend == 2) {
    EDIT_TRY(flush_small());
  } else if (npend == 1) {
    EDIT_TRY(q.decide(pend_layer[0]));
    EDIT_TRY(flush_pass2());
  }
  return q.finish_round(layers, count);
}

}  // extern "C"

namespace {

// Page-locked host memory (hipHostMalloc, or torch's pin_memory), which the
// copy engines can read and write asynchronously.
bool is_pinned_host(const void* p) {
  hipPointerAttribute_t attr;
  const hipError_t e = hipPointerGetAttributes(&attr, p);
  if (e != hipSuccess) {
    (void)hipGetLastError();  // an unregistered pointer is an answer, not a failure
    return false;
  }
  return attr.type == hipMemoryTypeHost;
}

edit_status_t offload_setup(edit_outer* h) {
  Offload& o = h->off;
  if (o.ready) return EDIT_OK;
  int64_t cap = 64;
  for (const Unit& u : h->units) cap = std::max(cap, u.n);
  cap = ceil_div(cap, 64) * 64;  // each half of a slot stays 256-byte aligned
  hipError_t e = hipMalloc(reinterpret_cast<void**>(&o.buf),
                           sizeof(float) * 2 * kOffloadSlots * static_cast<size_t>(cap));
  if (e != hipSuccess) {
    o.buf = nullptr;
    return fail(EDIT_ENOMEM, std::string("hipMalloc of the staging ring: ") + hipGetErrorString(e));
  }
  o.cap = cap;
  if ((e = hipStreamCreateWithFlags(&o.h2d, hipStreamNonBlocking)) != hipSuccess ||
      (e = hipStreamCreateWithFlags(&o.d2h, hipStreamNonBlocking)) != hipSuccess ||
      (e = hipEventCreateWithFlags(&o.start, hipEventDisableTiming)) != hipSuccess) {
    destroy_offload(h);
    return fail_hip(e, "offload streams");
  }
  for (int s = 0; s < kOffloadSlots; ++s)
    if ((e = hipEventCreateWithFlags(&o.in_done[s], hipEventDisableTiming)) != hipSuccess ||
        (e = hipEventCreateWithFlags(&o.comp_done[s], hipEventDisableTiming)) != hipSuccess ||
        (e = hipEventCreateWithFlags(&o.out_done[s], hipEventDisableTiming)) != hipSuccess) {
      destroy_offload(h);
      return fail_hip(e, "offload events");
    }
  o.ready = true;
  return EDIT_OK;
}

}  // namespace

extern "C" {

edit_status_t edit_outer_step_round_host(edit_outer_t h, int32_t count, const int32_t* layers,
                                         float* const* theta_host, float* const* momentum_host,
                                         void* const* replicas, void* stream) {
  if (!h) return fail(EDIT_EINVAL, "NULL handle");
  if (count < 1) return fail(EDIT_EINVAL, "count must be >= 1");
  if (!layers || !theta_host || !momentum_host || !replicas)
    return fail(EDIT_EINVAL, "layers, theta_host, momentum_host and replicas must not be NULL");
  EDIT_TRY(check_device(h));
  EDIT_TRY(offload_setup(h));
  Offload& o = h->off;
  const int K = h->cfg.num_workers;
  std::vector<char> seen(h->cfg.num_layers, 0);
  for (int32_t i = 0; i < count; ++i) {
    const int32_t l = layers[i];
    // the replicas are checked against a staging slot standing in for theta/b
    EDIT_TRY(check_step(h, l, o.buf, o.buf + o.cap, replicas + static_cast<size_t>(i) * K));
    if (seen[l]++) return fail(EDIT_EINVAL, "layer " + std::to_string(l) + " appears twice in a round");
    const int64_t n = h->units[l].n;
    if (n == 0) continue;
    const float* th = theta_host[i];
    const float* mo = momentum_host[i];
    if (!th || !mo) return fail(EDIT_EINVAL, "theta_host and momentum_host must not be NULL");
    if (!is_pinned_host(th) || !is_pinned_host(mo))
      return fail(EDIT_EINVAL, "theta_host and momentum_host of layer " + std::to_string(l) +
                                   " must be pinned host memory (hipHostMalloc)");
    const uintptr_t a = reinterpret_cast<uintptr_t>(th), b = reinterpret_cast<uintptr_t>(mo);
    if (a < b + 4 * n && b < a + 4 * n)
      return fail(EDIT_EINVAL, "theta_host and momentum_host overlap");
  }
  hipStream_t cs = reinterpret_cast<hipStream_t>(stream);
  Enqueue q{h, cs, decide_params(h), K, h->cfg.replica_dtype == EDIT_BF16};
  hipError_t e = hipEventRecord(o.start, cs);
  if (e == hipSuccess) e = hipStreamWaitEvent(o.h2d, o.start, 0);
  if (e != hipSuccess) return fail_hip(e, "round start");
  bool used_now[kOffloadSlots] = {};
  for (int32_t i = 0; i < count; ++i) {
    const int32_t l = layers[i];
    Unit& u = h->units[l];
    const int s = i % kOffloadSlots;
    float* dth = o.buf + static_cast<size_t>(s) * 2 * o.cap;
    float* db = dth + o.cap;
    void* const* reps = replicas + static_cast<size_t>(i) * K;
    const size_t bytes = sizeof(float) * static_cast<size_t>(u.n);
    // copy in, once the slot's previous unit has been copied out
    if (o.used[s] && (e = hipStreamWaitEvent(o.h2d, o.out_done[s], 0)) != hipSuccess)
      return fail_hip(e, "hipStreamWaitEvent");
    if (u.n > 0 &&
        ((e = hipMemcpyAsync(dth, theta_host[i], bytes, hipMemcpyHostToDevice, o.h2d)) != hipSuccess ||
         (e = hipMemcpyAsync(db, momentum_host[i], bytes, hipMemcpyHostToDevice, o.h2d)) != hipSuccess))
      return fail_hip(e, "copy to device");
    if ((e = hipEventRecord(o.in_done[s], o.h2d)) != hipSuccess ||
        (e = hipStreamWaitEvent(cs, o.in_done[s], 0)) != hipSuccess)
      return fail_hip(e, "copy-in event");
    // the step itself, on the caller's stream, from the staging slot
    EDIT_TRY(q.event(u, l, 0));
    if (h->one_pass) {
      EDIT_TRY(q.fused(l, dth, db, reps));
      EDIT_TRY(q.event(u, l, 1));
      EDIT_TRY(q.event(u, l, 2));
      EDIT_TRY(q.records(l, 1));
    } else {
      EDIT_TRY(q.pass1(l, dth, reps, nullptr));
      EDIT_TRY(q.decide(l));
      EDIT_TRY(q.event(u, l, 1));
      EDIT_TRY(q.event(u, l, 2));
      EDIT_TRY(q.pass2(l, dth, db, reps));
    }
    EDIT_TRY(q.event(u, l, 3));
    // copy out once the step is done
    if ((e = hipEventRecord(o.comp_done[s], cs)) != hipSuccess ||
        (e = hipStreamWaitEvent(o.d2h, o.comp_done[s], 0)) != hipSuccess)
      return fail_hip(e, "compute event");
    if (u.n > 0 &&
        ((e = hipMemcpyAsync(theta_host[i], dth, bytes, hipMemcpyDeviceToHost, o.d2h)) != hipSuccess ||
         (e = hipMemcpyAsync(momentum_host[i], db, bytes, hipMemcpyDeviceToHost, o.d2h)) != hipSuccess))
      return fail_hip(e, "copy to host");
    if ((e = hipEventRecord(o.out_done[s], o.d2h)) != hipSuccess) return fail_hip(e, "copy-out event");
    o.used[s] = true;
    used_now[s] = true;
  }
  // the caller's stream covers the copies back: synchronising it makes the
  // host arrays current
  for (int s = 0; s < kOffloadSlots; ++s)
    if (used_now[s] && (e = hipStreamWaitEvent(cs, o.out_done[s], 0)) != hipSuccess)
      return fail_hip(e, "round end");
  return q.finish_round(layers, count);
}

edit_status_t edit_outer_state_get(edit_outer_t h, int32_t layer, edit_layer_state_t* out) {
  if (!h || !out) return fail(EDIT_EINVAL, "NULL argument");
  if (layer < 0 || layer >= h->cfg.num_layers)
    return fail(EDIT_EINVAL, "layer " + std::to_string(layer) + " out of range");
  Unit& u = h->units[layer];
  if (!u.has_state) return fail(EDIT_ESTATE, "unit has neither stepped nor had its state set");
  edit_status_t st = check_device(h);
  if (st != EDIT_OK) return st;
  EDIT_TRY(wait_unit(h, u));
  hipError_t e = hipSuccess;
  UnitRecord rec;
  if ((e = hipMemcpy(&rec, u.rec, sizeof rec, hipMemcpyDeviceToHost)) != hipSuccess)
    return fail_hip(e, "hipMemcpy D2H");
  std::memset(out, 0, sizeof *out);
  const int K = h->cfg.num_workers;
  out->round = rec.round;
  out->num_workers = K;
  out->rolled_back = rec.rollback;
  out->z_tested = rec.z_tested;
  for (int j = 0; j < K; ++j) {
    out->ema_mean[j] = rec.mu[j];
    out->ema_std[j] = rec.sigma[j];
    out->norm[j] = rec.norm[j];
    out->weight[j] = rec.weight[j];
    out->anomalous[j] = rec.anomalous[j];
  }
  out->synced_norm = rec.synced_norm;
  out->clip_coef = rec.clip_coef;
  return EDIT_OK;
}

edit_status_t edit_outer_state_set(edit_outer_t h, int32_t layer, const edit_layer_state_t* in) {
  if (!h || !in) return fail(EDIT_EINVAL, "NULL argument");
  if (layer < 0 || layer >= h->cfg.num_layers)
    return fail(EDIT_EINVAL, "layer " + std::to_string(layer) + " out of range");
  if (in->round < 0) return fail(EDIT_EINVAL, "round must be >= 0");
  const int K = h->cfg.num_workers;
  for (int j = 0; j < K; ++j)
    if (!std::isfinite(in->ema_mean[j]) || !(in->ema_std[j] >= 0.0) || !std::isfinite(in->ema_std[j]))
      return fail(EDIT_EINVAL, "EMA state must be finite with ema_std >= 0");
  Unit& u = h->units[layer];
  edit_status_t st = check_device(h);
  if (st != EDIT_OK) return st;
  EDIT_TRY(wait_unit(h, u));
  hipError_t e = hipSuccess;
  UnitRecord rec;
  if ((e = hipMemcpy(&rec, u.rec, sizeof rec, hipMemcpyDeviceToHost)) != hipSuccess)
    return fail_hip(e, "hipMemcpy D2H");
  for (int j = 0; j < K; ++j) {
    rec.mu[j] = in->ema_mean[j];
    rec.sigma[j] = in->ema_std[j];
  }
  rec.round = in->round;
  rec.stepped = 1;
  if ((e = hipMemcpy(u.rec, &rec, sizeof rec, hipMemcpyHostToDevice)) != hipSuccess)
    return fail_hip(e, "hipMemcpy H2D");
  u.has_state = true;
  return EDIT_OK;
}

void edit_outer_destroy(edit_outer_t h) {
  if (!h) return;
  int prev = -1;
  if (hipGetDevice(&prev) == hipSuccess && prev != h->device) (void)hipSetDevice(h->device);
  for (Unit& u : h->units) (void)wait_unit(h, u);
  destroy_units(h);
  if (prev >= 0 && prev != h->device) (void)hipSetDevice(prev);
  delete h;
}

edit_status_t edit_outer_set_profiling(edit_outer_t h, int32_t every) {
  if (!h) return fail(EDIT_EINVAL, "NULL handle");
  if (every < 0) return fail(EDIT_EINVAL, "every must be >= 0");
  h->profile_every = every;
  return EDIT_OK;
}

edit_status_t edit_outer_kernel_times(edit_outer_t h, int32_t layer, float ms[2]) {
  if (!h || !ms) return fail(EDIT_EINVAL, "NULL argument");
  if (layer < 0 || layer >= h->cfg.num_layers)
    return fail(EDIT_EINVAL, "layer " + std::to_string(layer) + " out of range");
  Unit& u = h->units[layer];
  if (!u.profiled) return fail(EDIT_ESTATE, "the unit's last step was not profiled");
  hipError_t e = hipEventSynchronize(u.prof[3]);
  if (e != hipSuccess) return fail_hip(e, "hipEventSynchronize");
  if ((e = hipEventElapsedTime(&ms[0], u.prof[0], u.prof[1])) != hipSuccess ||
      (e = hipEventElapsedTime(&ms[1], u.prof[2], u.prof[3])) != hipSuccess)
    return fail_hip(e, "hipEventElapsedTime");
  return EDIT_OK;
}

edit_status_t edit_outer_update_probe(edit_outer_t h, int32_t layer, float* theta, float* momentum,
                                      void* const* replicas, void* stream) {
  if (!h) return fail(EDIT_EINVAL, "NULL handle");
  EDIT_TRY(check_step(h, layer, theta, momentum, replicas));
  EDIT_TRY(check_device(h));
  const Unit& u = h->units[layer];
  if (u.n == 0) return EDIT_OK;
  const hipError_t e =
      launch_pattern_probe(h->cfg.num_workers, h->cfg.replica_dtype == EDIT_BF16, u.blocks2, h->pass2_lds, theta,
                           momentum, replicas, u.n, reinterpret_cast<hipStream_t>(stream));
  return e == hipSuccess ? EDIT_OK : fail_hip(e, "update probe launch");
}

edit_status_t edit_outer_copy_probe(void* dst, const void* src, int64_t nbytes, void* stream) {
  if (nbytes < 0 || (nbytes & 15)) return fail(EDIT_EINVAL, "nbytes must be a non-negative multiple of 16");
  if (nbytes == 0) return EDIT_OK;
  if (!dst || !src || !aligned16(dst) || !aligned16(src))
    return fail(EDIT_EINVAL, "dst and src must be non-NULL and 16-byte aligned");
  const uintptr_t d = reinterpret_cast<uintptr_t>(dst), s = reinterpret_cast<uintptr_t>(src);
  if (d < s + nbytes && s < d + nbytes) return fail(EDIT_EINVAL, "dst and src overlap");
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail_hip(e, "hipGetDevice");
  // One 16-byte vector per thread, a flat grid, as in the update pass (a
  // persistent grid-stride copy measured 4.6 TB/s against 6.2 here); the
  // grid-stride loop only takes over past the largest grid.
  const int64_t nvec = nbytes / 16;
  const int blocks = static_cast<int>(std::max<int64_t>(1, std::min<int64_t>(INT32_MAX, ceil_div(nvec, kThreads))));
  e = launch_copy(dst, src, nbytes, blocks, reinterpret_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail_hip(e, "copy launch");
  return EDIT_OK;
}

}  // extern "C"
