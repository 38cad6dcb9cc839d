// Internal declarations of the sync-group worker path (one rank of a group
// whose K replicas sit on K GPUs), shared by edit_group_kernels.hip and
// edit_group_runtime.hip.  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "edit_outer.h"

namespace edit {

constexpr int kGroupThreads = 256;        // streaming passes
constexpr int kGroupNormVecs = 2;        // 16-byte vectors per thread of the norm pass
constexpr int kGroupUpdateThreads = 128;  // the update pass
constexpr int kGroupOneBlock = 1024;      // the one-block reductions

// Device-resident state and decision of one unit on one rank.
struct alignas(16) GroupRecord {
  double mu, sigma;               // this worker's EMA pair (Eq. 1)
  double self_norm;               // G_rank of the last step
  double norm[EDIT_MAX_K];        // every worker's G_j, from the all-gather
  double weight[EDIT_MAX_K];      // w_j
  double synced_norm;             // ||Delta_bar||
  double clip_coef;               // beta
  int64_t round;                  // completed rounds of this unit
  int32_t self_flag;              // this worker failed the z-test (or G is not finite)
  int32_t rollback;               // every worker flagged
  int32_t z_tested;
  int32_t stepped;
  uint8_t anomalous[EDIT_MAX_K];
};

struct GroupParams {
  double alpha, delta, phi, eps;
  int64_t warmup;
  uint32_t flags;
};

hipError_t launch_group_norm(bool bf16, int rows, const float* theta, const void* rep, float* delta,
                             int64_t n, double* partials, hipStream_t stream);
hipError_t launch_group_self(const double* partials, int rows, GroupRecord* rec, double* norm_out,
                             const GroupParams& prm, hipStream_t stream);
// `blocks` blocks: block 0 takes the decision; all of them clear `delta`
// when this worker is flagged.
hipError_t launch_group_weights(int blocks, const double* gathered, int K, int rank, GroupRecord* rec,
                                double* weight_out, float* delta, int64_t n, const GroupParams& prm,
                                hipStream_t stream);
hipError_t launch_group_dbar(int rows, const GroupRecord* rec, const float* dbar, int64_t n,
                             double* partials, hipStream_t stream);
hipError_t launch_group_clip(const double* partials, int rows, GroupRecord* rec, const GroupParams& prm,
                             hipStream_t stream);
hipError_t launch_group_update(bool bf16, int blocks, const GroupRecord* rec, const float* dbar,
                               float* theta, float* mom, void* rep, int64_t n, double lr, double rho,
                               hipStream_t stream);
int group_dbar_blocks_per_cu();

// Shared with the single-GPU runtime (edit_outer_runtime.hip): the calling
// thread's last-error message, the configuration checks of edit_outer_init,
// and the current device if it is a gfx950 (its index and CU count).
edit_status_t set_error(edit_status_t s, const char* msg);
edit_status_t validate_config(const edit_outer_config_t* cfg);
edit_status_t current_gfx950(int* device, int* num_cu);

}  // namespace edit
