// Launchers of the outer-step kernels by worker count K: each call finds the
// kernel set of K's range (one object of edit_outer_kernels.hip per range)
// and forwards to it.  Host code only.
#include "edit_outer_internal.h"

namespace edit {
namespace {

const KernelSet* kernels_for(int K) {
#define EDIT_RANGE(first, last) \
  if (K >= (first) && K <= (last)) return EDIT_KERNEL_SET_FN(first)(K);
  EDIT_K_RANGES(EDIT_RANGE)
#undef EDIT_RANGE
  return nullptr;
}

}  // namespace

hipError_t launch_pass1(int K, bool bf16, int rows, const float* theta, const void* const* reps,
                        int64_t n, double* partials, const double* prev_partials, int prev_rows,
                        UnitRecord* prev_rec, const DecideParams& prm, hipStream_t stream) {
  const KernelSet* s = kernels_for(K);
  return s ? s->pass1(bf16, rows, theta, reps, n, partials, prev_partials, prev_rows, prev_rec, prm, stream)
           : hipErrorInvalidValue;
}

hipError_t launch_pass1_pair(int K, bool bf16, const Pass1Desc* unit, int count, const DecideDesc* prev,
                             int nprev, const DecideParams& prm, hipStream_t stream) {
  if (count < 1 || count > 2 || nprev < 0 || nprev > 2) return hipErrorInvalidValue;
  const KernelSet* s = kernels_for(K);
  return s ? s->pass1_pair(bf16, unit, count, prev, nprev, prm, stream) : hipErrorInvalidValue;
}

hipError_t launch_round_small(int K, bool bf16, const DecideDesc* prev, int nprev, const DecideParams& prm,
                              const SingleBlockDesc* unit, int count, double lr, double rho,
                              hipStream_t stream) {
  if (count < 0 || count > kMaxSingleBlockUnits || nprev < 0 || nprev > 2) return hipErrorInvalidValue;
  const KernelSet* s = kernels_for(K);
  return s ? s->round_small(bf16, prev, nprev, prm, unit, count, lr, rho, stream) : hipErrorInvalidValue;
}

hipError_t launch_decide(int K, const double* partials, int rows, UnitRecord* rec, const DecideParams& prm,
                         hipStream_t stream) {
  const KernelSet* s = kernels_for(K);
  return s ? s->decide(partials, rows, rec, prm, stream) : hipErrorInvalidValue;
}

hipError_t launch_gram_reduce(int K, const double* partials, int rows, double* gram, hipStream_t stream) {
  const KernelSet* s = kernels_for(K);
  return s ? s->gram_reduce(partials, rows, gram, stream) : hipErrorInvalidValue;
}

hipError_t launch_decide_gram(int K, const double* gram, UnitRecord* rec, const DecideParams& prm,
                              hipStream_t stream) {
  const KernelSet* s = kernels_for(K);
  return s ? s->decide_gram(gram, rec, prm, stream) : hipErrorInvalidValue;
}

hipError_t launch_pass2(int K, bool bf16, int blocks, int lds, float* theta, float* mom, void* const* reps,
                        const UnitRecord* rec, int64_t n, double lr, double rho, hipStream_t stream) {
  const KernelSet* s = kernels_for(K);
  return s ? s->pass2(bf16, blocks, lds, theta, mom, reps, rec, n, lr, rho, stream) : hipErrorInvalidValue;
}

// The update pass streams 2K + 4 buffers at once (K + 2 read, K + 2
// written), and the HBM serves that mix faster with fewer of its waves in
// flight than its registers allow.  Sweeps on one box (alternating runs,
// 1B round at K = 8 bf16): 128-thread blocks, 8 per CU (the register
// limit) 14.31-14.36 ms, 4 per CU 13.91-14.01, 3 per CU 13.84-13.87;
// one-wave blocks, 6 per CU 13.56-13.60 ms, against 13.60-13.68 at 4 or 5,
// 13.72-13.73 at 7 and 14.00-14.02 at 8.  Six one-wave blocks per CU also
// gave the shortest 350M, 7B half-shard and A-EDiT K = 16 rounds.
int update_pass_blocks_per_cu(int K) {
  (void)K;
  return 6;
}

int update_pass_lds(int K, int lds_per_cu) {
  // the largest multiple of 256 bytes that still lets that many blocks fit
  return lds_per_cu > 0 ? (lds_per_cu / update_pass_blocks_per_cu(K)) & ~255 : 0;
}

int fused_vectors_per_thread(int K, bool bf16) {
  const KernelSet* s = kernels_for(K);
  return s ? (bf16 ? s->fused_vectors_bf16 : s->fused_vectors_f32) : 1;
}

// The one-pass kernel streams the same 2K + 4 buffers as the update pass.
// With bf16 replicas (two 16-byte vectors per thread) and one-wave blocks,
// six resident blocks per CU measured best at the 1B shape (rocprofv3, A/B
// runs on one box): 435 us per unit against 438-442 at five or seven blocks
// and 441 for 128-thread blocks at four per CU (the earlier shape, itself
// 10.64-10.73 ms per round against 11.02-11.07 uncapped).  One vector per
// thread took 474-484 us: each block's closing reduction and partial row
// then cover half as much data.  Other cases keep the occupancy their
// registers give.
int one_pass_lds(int K, bool bf16, int lds_per_cu) {
  const int blocks = bf16 && K <= 16 ? 6 : 0;
  return blocks > 0 && lds_per_cu > 0 ? (lds_per_cu / blocks) & ~255 : 0;
}

hipError_t launch_fused_mean(int K, bool bf16, int rows, int lds, float* theta, float* mom, void* const* reps,
                             double* partials, UnitRecord* rec, int64_t n, double lr, double rho,
                             hipStream_t stream) {
  const KernelSet* s = kernels_for(K);
  return s ? s->fused_mean(bf16, rows, lds, theta, mom, reps, partials, rec, n, lr, rho, stream)
           : hipErrorInvalidValue;
}

hipError_t launch_fused_finish(int K, const FinishEntry* table, int units, hipStream_t stream) {
  const KernelSet* s = kernels_for(K);
  return s ? s->fused_finish(table, units, stream) : hipErrorInvalidValue;
}

hipError_t launch_pattern_probe(int K, bool bf16, int blocks, int lds, float* theta, float* mom, void* const* reps,
                                int64_t n, hipStream_t stream) {
  const KernelSet* s = kernels_for(K);
  return s ? s->pattern_probe(bf16, blocks, lds, theta, mom, reps, n, stream) : hipErrorInvalidValue;
}

int pass1_blocks_per_cu(int K, bool bf16) {
  const KernelSet* s = kernels_for(K);
  return s ? s->pass1_blocks_per_cu(bf16) : 1;
}

}  // namespace edit
