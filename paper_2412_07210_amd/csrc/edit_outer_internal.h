// Internal declarations shared by the kernels and the host runtime of
// libedit_outer.so.  Not part of the public ABI (include/edit_outer.h).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "edit_outer.h"

namespace edit {

constexpr int kThreads = 256;        // threads per block of the Gram pass
constexpr int kPass2Threads = 64;    // threads per block of the update pass (one wave)
constexpr int kFusedThreads = 64;    // threads per block of the one-pass mean step (one wave)
constexpr int kMaxK = EDIT_MAX_K;
constexpr int kMaxPairs = kMaxK * (kMaxK + 1) / 2;

// Device-resident state and decision of one sync unit.  Written by the
// decision kernel, read by the update pass and copied out by state_get.
struct alignas(16) UnitRecord {
  double mu[kMaxK];         // EMA mean of G_j (Eq. 1)
  double sigma[kMaxK];      // EMA std of G_j (Eq. 1)
  double norm[kMaxK];       // G_j of the last step
  double weight[kMaxK];     // w_j of the last step
  double synced_norm;       // ||Delta_bar||
  double clip_coef;         // beta
  int64_t round;            // completed rounds of this unit
  double coef[kMaxK];       // beta * w_j, consumed by the update pass
  int32_t src[kMaxK];       // worker whose data the update pass loads for slot j
  int32_t rollback;         // 1: every worker flagged, reset replicas only
  int32_t use_deltas;       // 0: no worker has a non-zero coefficient
  int32_t z_tested;
  int32_t stepped;          // at least one step or state_set happened
  int32_t finish_pending;   // one-pass mode: partials written, record not yet made
  uint8_t anomalous[kMaxK];
};

// Where the one-pass record reduction of a unit finds its inputs.
struct FinishEntry {
  const double* partials;
  UnitRecord* rec;
  int32_t rows;
  int32_t pad;
};

struct DecideParams {
  double alpha, delta, phi, eps;
  int64_t warmup;
  uint32_t flags;
};

// A unit of a round whose Gram pass is a single block, stepped whole (Gram
// row, decision, update) by one block of a small launch.
constexpr int kMaxSingleBlockUnits = 4;  // per launch
struct SingleBlockDesc {
  float* theta;
  float* mom;
  void* const* reps;  // host array of K device pointers (read at launch)
  double* partials;
  UnitRecord* rec;
  int64_t n;
};

// A unit whose decision block 0 of a launch takes (see launch_pass1_pair).
struct DecideDesc {
  const double* partials;
  int rows;
  UnitRecord* rec;
};

// One unit of a two-unit Gram launch.
struct Pass1Desc {
  const float* theta;
  const void* const* reps;  // host array of K device pointers (read at launch)
  int64_t n;
  double* partials;
  int rows;
};

// The kernels specialised for one K, behind plain function pointers.  The
// kernels file is compiled once per range of K below (the ranges' template
// instantiations then compile in parallel); the object of the range that
// starts at F exports EDIT_KERNEL_SET_FN(F)(K), which returns the set of a K
// in its range and nullptr otherwise.
#define EDIT_K_RANGES(X) X(1, 8) X(9, 16) X(17, 24) X(25, 32)
#define EDIT_KERNEL_SET_FN2(first) kernel_set_from_##first
#define EDIT_KERNEL_SET_FN(first) EDIT_KERNEL_SET_FN2(first)

struct KernelSet {
  hipError_t (*pass1)(bool bf16, int rows, const float* theta, const void* const* reps, int64_t n,
                      double* partials, const double* prev_partials, int prev_rows, UnitRecord* prev_rec,
                      const DecideParams& prm, hipStream_t stream);
  hipError_t (*pass1_pair)(bool bf16, const Pass1Desc* unit, int count, const DecideDesc* prev, int nprev,
                           const DecideParams& prm, hipStream_t stream);
  hipError_t (*round_small)(bool bf16, const DecideDesc* prev, int nprev, const DecideParams& prm,
                            const SingleBlockDesc* unit, int count, double lr, double rho, hipStream_t stream);
  hipError_t (*decide)(const double* partials, int rows, UnitRecord* rec, const DecideParams& prm,
                       hipStream_t stream);
  hipError_t (*gram_reduce)(const double* partials, int rows, double* gram, hipStream_t stream);
  hipError_t (*decide_gram)(const double* gram, UnitRecord* rec, const DecideParams& prm, hipStream_t stream);
  hipError_t (*pass2)(bool bf16, int blocks, int lds, float* theta, float* mom, void* const* reps,
                      const UnitRecord* rec, int64_t n, double lr, double rho, hipStream_t stream);
  hipError_t (*fused_mean)(bool bf16, int rows, int lds, float* theta, float* mom, void* const* reps,
                           double* partials, UnitRecord* rec, int64_t n, double lr, double rho, hipStream_t stream);
  hipError_t (*fused_finish)(const FinishEntry* table, int units, hipStream_t stream);
  int (*pass1_blocks_per_cu)(bool bf16);
  hipError_t (*pattern_probe)(bool bf16, int blocks, int lds, float* theta, float* mom, void* const* reps,
                              int64_t n, hipStream_t stream);
  int fused_vectors_bf16, fused_vectors_f32;
};

#define EDIT_DECLARE_SET(first, last) const KernelSet* EDIT_KERNEL_SET_FN(first)(int K);
EDIT_K_RANGES(EDIT_DECLARE_SET)
#undef EDIT_DECLARE_SET

// Launchers (edit_outer_dispatch.hip, through the kernel sets).  All enqueue
// on `stream` and return the launch status (hipErrorInvalidValue for a K
// outside 1..EDIT_MAX_K); none synchronises.
// Pass 1 over `rows` partial rows; when prev_partials is not null, one more
// block takes the decision of the previous unit of a round (prev_rows rows,
// record prev_rec) inside the same launch.
hipError_t launch_pass1(int K, bool bf16, int rows, const float* theta,
                        const void* const* reps, int64_t n, double* partials,
                        const double* prev_partials, int prev_rows, UnitRecord* prev_rec,
                        const DecideParams& prm, hipStream_t stream);
// Pass 1 of `count` (1 or 2) units of a round in one launch, K <= 8 only:
// each block writes its row of every unit (the rows of its own launch), and
// block 0 takes the decisions of `nprev` (0 to 2) earlier units first.
hipError_t launch_pass1_pair(int K, bool bf16, const Pass1Desc* unit, int count, const DecideDesc* prev,
                             int nprev, const DecideParams& prm, hipStream_t stream);
// A small launch of a round: the decisions of `nprev` (0 to 2) earlier
// units and `count` whole single-block units.
hipError_t launch_round_small(int K, bool bf16, const DecideDesc* prev, int nprev, const DecideParams& prm,
                              const SingleBlockDesc* unit, int count, double lr, double rho,
                              hipStream_t stream);
hipError_t launch_decide(int K, const double* partials, int rows, UnitRecord* rec,
                         const DecideParams& prm, hipStream_t stream);
// The fixed-order sum of the partials as a K(K+1)/2 vector in device memory.
hipError_t launch_gram_reduce(int K, const double* partials, int rows, double* gram,
                              hipStream_t stream);
// The decision from a device-resident Gram vector.
hipError_t launch_decide_gram(int K, const double* gram, UnitRecord* rec, const DecideParams& prm,
                              hipStream_t stream);
// The update pass; `lds` bytes of dynamic LDS per block (used by nothing)
// cap its resident blocks per CU (update_pass_lds).
hipError_t launch_pass2(int K, bool bf16, int blocks, int lds, float* theta, float* mom,
                        void* const* reps, const UnitRecord* rec, int64_t n, double lr,
                        double rho, hipStream_t stream);
// Update-pass blocks resident per CU, and the dynamic LDS per block that
// caps them there given the CU's LDS bytes.
int update_pass_blocks_per_cu(int K);
int update_pass_lds(int K, int lds_per_cu);
// One-pass mean step (no penalty components): `rows` blocks of
// fused_vectors_per_thread(K, bf16) * kFusedThreads vectors each, leaving
// rows x (K+1) norm partials (each block's K+1 sums contiguous) and the unit marked; then one block per entry
// of `table` turns marked units' partials into their records.
int fused_vectors_per_thread(int K, bool bf16);
// `lds`: dynamic LDS per block capping its resident blocks per CU
// (one_pass_lds), as for the update pass.
int one_pass_lds(int K, bool bf16, int lds_per_cu);
hipError_t launch_fused_mean(int K, bool bf16, int rows, int lds, float* theta, float* mom,
                             void* const* reps, double* partials, UnitRecord* rec, int64_t n,
                             double lr, double rho, hipStream_t stream);
hipError_t launch_fused_finish(int K, const FinishEntry* table, int units, hipStream_t stream);
hipError_t launch_copy(void* dst, const void* src, int64_t nbytes, int blocks,
                       hipStream_t stream);
// Pass 2's loads and stores (whole vectors only) with no arithmetic.
hipError_t launch_pattern_probe(int K, bool bf16, int blocks, int lds, float* theta, float* mom, void* const* reps,
                                int64_t n, hipStream_t stream);

// Resident blocks per CU of the pass-1 kernel (for its persistent grid).
int pass1_blocks_per_cu(int K, bool bf16);

inline int num_pairs(int K) { return K * (K + 1) / 2; }

}  // namespace edit
