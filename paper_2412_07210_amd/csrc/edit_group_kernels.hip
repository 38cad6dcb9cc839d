// Device kernels of one worker of an EDiT sync group on its own GPU.
//
// In EDiT a module's K replicas sit on the K workers of a model sync group,
// each running the Sync() procedure (appendix, Algorithm 2) on its own copy.
// One worker (rank) of that layout runs, per sync unit:
//
//   group_norm      streams theta and its own replica once: the exact fp64
//                   pseudo gradient's squared norm, per-block partials, and
//                   Delta exported in fp32 for the group's all-reduce;
//   group_self      one block: the fixed-order sum of those partials, G_rank,
//                   the z-test and EMA update of this worker (Eq. 1), and the
//                   pair {G_rank, flag} for the group's all-gather;
//   group_weights   the first wave of block 0: the decision of all K workers from the gathered
//                   pairs (mask, rollback, softmax weights of Eq. 2), the same
//                   on every rank; in the same launch a flagged worker's
//                   export is set to zero, so its (possibly non-finite)
//                   pseudo gradient never enters the sum;
//   group_dbar      streams the all-reduced Delta_bar: per-block partials of
//                   its squared norm;
//   group_clip      one block: Gbar and beta (Eq. 4);
//   group_update    Delta_hat = beta*Delta_bar, Nesterov (OuterOpt) on theta
//                   and b, and the own replica set to theta' (the rollback
//                   branch sets it to theta only).
//
// Arithmetic is fp64 as in the single-GPU step; the exported Delta and the
// all-reduced Delta_bar are fp32 (the payload of the collective).  All
// reductions run in a fixed order, so a rank's results are reproducible.
#include "edit_group_internal.h"

namespace edit {
namespace {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float float2_t __attribute__((ext_vector_type(2)));

template <bool BF16>
struct GVec {
  static constexpr int VE = BF16 ? 8 : 4;  // elements per 16-byte replica vector
};

template <bool NT, typename T>
__device__ __forceinline__ T gld(const T* p) {
  if constexpr (NT)
    return __builtin_nontemporal_load(p);
  else
    return *p;
}
template <bool NT, typename T>
__device__ __forceinline__ void gst(T* p, T v) {
  if constexpr (NT)
    __builtin_nontemporal_store(v, p);
  else
    *p = v;
}

// Element e of a 16-byte replica vector, widened to fp32 (exact).
template <bool BF16>
__device__ __forceinline__ float gelem(const u32x4& raw, int e) {
  if constexpr (BF16) {
    const uint32_t word = raw[e >> 1];
    return __uint_as_float((e & 1) ? (word & 0xffff0000u) : (word << 16));
  } else {
    return __uint_as_float(raw[e]);
  }
}

template <bool BF16>
__device__ __forceinline__ float gscalar(const void* base, int64_t i) {
  if constexpr (BF16)
    return __uint_as_float(static_cast<uint32_t>(reinterpret_cast<const uint16_t*>(base)[i]) << 16);
  else
    return reinterpret_cast<const float*>(base)[i];
}

__device__ __forceinline__ uint32_t gpack2(float a, float b) {
  const float2_t f = {a, b};
  const bf16x2_t h = __builtin_convertvector(f, bf16x2_t);  // RNE
  return __builtin_bit_cast(uint32_t, h);
}

template <bool BF16>
__device__ __forceinline__ void gstore_scalar(void* base, int64_t i, float x) {
  if constexpr (BF16)
    reinterpret_cast<uint16_t*>(base)[i] = static_cast<uint16_t>(gpack2(x, 0.f) & 0xffffu);
  else
    reinterpret_cast<float*>(base)[i] = x;
}

// VE fp32 values of a theta/momentum/delta buffer at vector v.
template <int VE, bool NT>
__device__ __forceinline__ void gload_f32(const float* p, int64_t v, float (&x)[VE]) {
  const f32x4* q = reinterpret_cast<const f32x4*>(p) + v * (VE / 4);
#pragma unroll
  for (int h = 0; h < VE / 4; ++h) {
    const f32x4 t = gld<NT>(q + h);
#pragma unroll
    for (int c = 0; c < 4; ++c) x[4 * h + c] = t[c];
  }
}

template <int VE, bool NT>
__device__ __forceinline__ void gstore_f32(float* p, int64_t v, const float (&x)[VE]) {
  f32x4* q = reinterpret_cast<f32x4*>(p) + v * (VE / 4);
#pragma unroll
  for (int h = 0; h < VE / 4; ++h) {
    f32x4 t;
#pragma unroll
    for (int c = 0; c < 4; ++c) t[c] = x[4 * h + c];
    gst<NT>(q + h, t);
  }
}

template <bool BF16>
__device__ __forceinline__ u32x4 gpack(const float (&x)[GVec<BF16>::VE]) {
  u32x4 r;
  if constexpr (BF16) {
#pragma unroll
    for (int c = 0; c < 4; ++c) r[c] = gpack2(x[2 * c], x[2 * c + 1]);
  } else {
#pragma unroll
    for (int c = 0; c < 4; ++c) r[c] = __float_as_uint(x[c]);
  }
  return r;
}

__device__ __forceinline__ double gwave_sum(double x) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) x += __shfl_xor(x, m, 64);
  return x;
}

// Sum of a block's per-thread values into one double, fixed order: wave
// butterflies, then the waves in order.  Every thread must call it.
template <int kBlock>
__device__ __forceinline__ double block_sum(double x) {
  __shared__ double red[kBlock / 64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  x = gwave_sum(x);
  if (lane == 0) red[wave] = x;
  __syncthreads();
  double s = red[0];
#pragma unroll
  for (int w = 1; w < kBlock / 64; ++w) s += red[w];
  return s;
}

// Fixed-order sum of `rows` partials by one block of kOneBlock threads:
// thread t takes rows t, t + kOneBlock, ..., then the block sum.
__device__ __forceinline__ double sum_partials(const double* partials, int rows) {
  double acc = 0.0;
  for (int r = threadIdx.x; r < rows; r += kGroupOneBlock) acc += partials[r];
  return block_sum<kGroupOneBlock>(acc);
}

// ------------------------------------------------------------- group_norm

template <bool BF16, bool NT>
__device__ __forceinline__ void gnorm_load(const float* theta, const void* rep, int64_t v, int64_t nvec,
                                           float (&th)[GVec<BF16>::VE], u32x4& raw) {
  if (v < nvec) {
    gload_f32<GVec<BF16>::VE, NT>(theta, v, th);
    raw = gld<NT>(reinterpret_cast<const u32x4*>(rep) + v);
  }
}

template <bool BF16, bool NT>
__device__ __forceinline__ void gnorm_vector(float* delta, int64_t v, int64_t nvec,
                                             const float (&th)[GVec<BF16>::VE], const u32x4& raw,
                                             double& acc) {
  constexpr int VE = GVec<BF16>::VE;
  if (v >= nvec) return;
  float out[VE];
#pragma unroll
  for (int e = 0; e < VE; ++e) {
    const double d = static_cast<double>(gelem<BF16>(raw, e)) - static_cast<double>(th[e]);
    acc = fma(d, d, acc);
    out[e] = static_cast<float>(d);
  }
  gstore_f32<VE, NT>(delta, v, out);
}

// A flat grid: each block owns kGroupNormVecs * kGroupThreads consecutive
// vectors, a thread loads its kGroupNormVecs vectors before computing, and
// the block leaves one partial sum of squares.  The pass writes 4 of every
// 10 bytes it moves (the fp32 export at bf16); with writes in the traffic a
// flat grid keeps the streams' in-flight window short and ordered (the
// update pass measured the same).
template <bool BF16, bool NT>
__global__ __launch_bounds__(kGroupThreads) void group_norm_kernel(const float* __restrict__ theta,
                                                                  const void* __restrict__ rep,
                                                                  float* __restrict__ delta,
                                                                  int64_t nvec, int64_t n,
                                                                  double* __restrict__ partials) {
  constexpr int VE = GVec<BF16>::VE;
  const int64_t v0 = static_cast<int64_t>(blockIdx.x) * (kGroupThreads * kGroupNormVecs) + threadIdx.x;
  float th[kGroupNormVecs][VE];
  u32x4 raw[kGroupNormVecs];
#pragma unroll
  for (int u = 0; u < kGroupNormVecs; ++u) {
    raw[u] = u32x4{0u, 0u, 0u, 0u};
    gnorm_load<BF16, NT>(theta, rep, v0 + u * kGroupThreads, nvec, th[u], raw[u]);
  }
  double acc = 0.0;
#pragma unroll
  for (int u = 0; u < kGroupNormVecs; ++u) gnorm_vector<BF16, NT>(delta, v0 + u * kGroupThreads, nvec, th[u], raw[u], acc);
  const int64_t i = nvec * VE + threadIdx.x;  // ragged tail: block 0
  if (blockIdx.x == 0 && i < n) {
    const double d = static_cast<double>(gscalar<BF16>(rep, i)) - static_cast<double>(theta[i]);
    acc = fma(d, d, acc);
    delta[i] = static_cast<float>(d);
  }
  const double s = block_sum<kGroupThreads>(acc);
  if (threadIdx.x == 0) partials[blockIdx.x] = s;
}

// ------------------------------------------------------------- group_self

// G_rank, this worker's z-test against its state before the round (no flag
// during the warm-up; a non-finite norm always flags), its EMA update when
// unflagged (Eq. 1), and the pair {G_rank, flag} for the all-gather.
__global__ __launch_bounds__(kGroupOneBlock) void group_self_kernel(const double* __restrict__ partials,
                                                                   int rows, GroupRecord* rec,
                                                                   double* __restrict__ norm_out,
                                                                   GroupParams prm) {
  const double ss = sum_partials(partials, rows);
  if (threadIdx.x != 0) return;
  const double G = sqrt(ss);
  const bool ae = prm.flags & EDIT_AE;
  const bool z_test = ae && rec->round >= prm.warmup;
  bool bad = !isfinite(G);
  const double mu0 = rec->mu, sg0 = rec->sigma;
  if (z_test && !bad) bad = (G - mu0) > prm.delta * sg0;
  if (ae && !bad) {
    const double mu = prm.alpha * G + (1.0 - prm.alpha) * mu0;
    const double dev = G - mu;
    rec->sigma = sqrt((1.0 - prm.alpha) * sg0 * sg0 + prm.alpha * dev * dev);
    rec->mu = mu;
  }
  rec->self_norm = G;
  rec->self_flag = bad ? 1 : 0;
  rec->z_tested = z_test ? 1 : 0;
  norm_out[0] = G;
  norm_out[1] = bad ? 1.0 : 0.0;
}

// ---------------------------------------------------------- group_weights

// The decision of the whole group from the gathered pairs, taken by the first
// wave of block 0 (worker j in lane j) in the same order on every rank: mask,
// rollback, weights (Eq. 2; the softmax of -G over the unflagged workers,
// shifted by their smallest norm), and this worker's weight for the
// all-reduce.  In the same launch every block clears its share of this
// worker's export when the worker was flagged by its own z-test (known from
// the earlier group_self launch), so its possibly non-finite pseudo gradient
// never enters the sum; otherwise those blocks return at once.
__global__ __launch_bounds__(kGroupThreads) void group_weights_kernel(const double* __restrict__ gathered, int K,
                                                                     int rank, GroupRecord* rec,
                                                                     double* __restrict__ weight_out,
                                                                     float* __restrict__ delta, int64_t n,
                                                                     GroupParams prm) {
  if (rec->self_flag) {  // grid-stride over 16-byte vectors, then the tail
    const int64_t nvec = n / 4;
    const int64_t stride = static_cast<int64_t>(gridDim.x) * kGroupThreads;
    const f32x4 z = {0.f, 0.f, 0.f, 0.f};
    for (int64_t v = static_cast<int64_t>(blockIdx.x) * kGroupThreads + threadIdx.x; v < nvec; v += stride)
      reinterpret_cast<f32x4*>(delta)[v] = z;
    const int64_t i = nvec * 4 + threadIdx.x;
    if (blockIdx.x == 0 && i < n) delta[i] = 0.f;
  }
  if (blockIdx.x != 0 || threadIdx.x >= 64) return;
  const int lane = threadIdx.x;
  const bool mine = lane < K;
  const double G = mine ? gathered[2 * lane] : 0.0;
  const bool flagged = mine ? (gathered[2 * lane + 1] != 0.0 || !isfinite(G)) : true;
  const bool ok = mine && !flagged;
  const int n_ok = __popcll(__ballot(ok));
  double w = 0.0;
  if (n_ok > 0) {
    if (prm.flags & EDIT_WA) {
      double g0 = ok ? G : INFINITY;
#pragma unroll
      for (int m = 32; m >= 1; m >>= 1) g0 = fmin(g0, __shfl_xor(g0, m, 64));
      const double e = ok ? exp(-(G - g0)) : 0.0;
      w = e / gwave_sum(e);
    } else {
      w = ok ? 1.0 / n_ok : 0.0;
    }
  }
  const double w_rank = __shfl(w, rank, 64);
  if (mine) {
    rec->norm[lane] = G;
    rec->anomalous[lane] = flagged ? 1 : 0;
    rec->weight[lane] = w;
  }
  if (lane == 0) {
    rec->rollback = n_ok == 0 ? 1 : 0;
    rec->round = rec->round + 1;
    rec->stepped = 1;
    rec->synced_norm = 0.0;
    rec->clip_coef = 0.0;
    weight_out[0] = w_rank;
  }
}

// ------------------------------------------------------------- group_dbar

// Squared norm of the all-reduced Delta_bar: persistent grid, per-block
// partials (nothing to do on a rollback).
template <bool NT>
__global__ __launch_bounds__(kGroupThreads) void group_dbar_kernel(const GroupRecord* __restrict__ rec,
                                                                  const float* __restrict__ dbar,
                                                                  int64_t n, double* __restrict__ partials) {
  if (rec->rollback) return;  // block-uniform
  const int64_t nvec = n / 4;
  const int64_t stride = static_cast<int64_t>(gridDim.x) * kGroupThreads;
  double acc = 0.0;
  for (int64_t v = static_cast<int64_t>(blockIdx.x) * kGroupThreads + threadIdx.x; v < nvec; v += stride) {
    const f32x4 x = gld<NT>(reinterpret_cast<const f32x4*>(dbar) + v);
#pragma unroll
    for (int c = 0; c < 4; ++c) acc = fma(static_cast<double>(x[c]), static_cast<double>(x[c]), acc);
  }
  const int64_t i = nvec * 4 + threadIdx.x;
  if (blockIdx.x == 0 && i < n) acc = fma(static_cast<double>(dbar[i]), static_cast<double>(dbar[i]), acc);
  const double s = block_sum<kGroupThreads>(acc);
  if (threadIdx.x == 0) partials[blockIdx.x] = s;
}

// Gbar = ||Delta_bar||, beta = min(phi / (Gbar + eps), 1) with the clip on.
__global__ __launch_bounds__(kGroupOneBlock) void group_clip_kernel(const double* __restrict__ partials,
                                                                   int rows, GroupRecord* rec,
                                                                   GroupParams prm) {
  if (rec->rollback) return;  // block-uniform
  const double ss = sum_partials(partials, rows);
  if (threadIdx.x != 0) return;
  const double gbar = sqrt(ss);
  rec->synced_norm = gbar;
  rec->clip_coef = (prm.flags & EDIT_GC) ? fmin(prm.phi / (gbar + prm.eps), 1.0) : 1.0;
}

// ----------------------------------------------------------- group_update

// theta' and b' of one element from Delta_hat (Sec. 4.1, as the single-GPU
// update pass): g = -Delta_hat; b' = rho b + g; theta' = theta - nu (g + rho b').
__device__ __forceinline__ void gnesterov(double dhat, float th, float b, double lr, double rho,
                                          float& th_out, float& b_out) {
  const double g = -dhat;
  const double bn = fma(rho, static_cast<double>(b), g);
  th_out = static_cast<float>(static_cast<double>(th) - lr * fma(rho, bn, g));
  b_out = static_cast<float>(bn);
}

// One 16-byte replica vector (and its theta, b, Delta_bar) per thread, blocks
// taken from the unit's end so the first ones find what group_dbar read last.
template <bool BF16, bool NT>
__global__ __launch_bounds__(kGroupUpdateThreads) void group_update_kernel(
    const GroupRecord* __restrict__ rec, const float* __restrict__ dbar, float* __restrict__ theta,
    float* __restrict__ mom, void* __restrict__ rep, int64_t nvec, int64_t n, double lr, double rho) {
  constexpr int VE = GVec<BF16>::VE;
  const int64_t v = static_cast<int64_t>(gridDim.x - 1 - blockIdx.x) * kGroupUpdateThreads + threadIdx.x;
  const int64_t tail = nvec * VE + threadIdx.x;
  const bool do_tail = blockIdx.x == 0 && tail < n;
  if (rec->rollback) {  // every worker flagged: the replica returns to theta_t
    if (v < nvec) {
      float th[VE];
      gload_f32<VE, NT>(theta, v, th);
      gst<NT>(reinterpret_cast<u32x4*>(rep) + v, gpack<BF16>(th));
    }
    if (do_tail) gstore_scalar<BF16>(rep, tail, theta[tail]);
    return;
  }
  const double beta = rec->clip_coef;
  if (v < nvec) {
    float th[VE], b[VE], d[VE], tn[VE], bn[VE];
    gload_f32<VE, NT>(theta, v, th);
    gload_f32<VE, NT>(mom, v, b);
    gload_f32<VE, NT>(dbar, v, d);
#pragma unroll
    for (int e = 0; e < VE; ++e) gnesterov(beta * static_cast<double>(d[e]), th[e], b[e], lr, rho, tn[e], bn[e]);
    gstore_f32<VE, NT>(theta, v, tn);
    gstore_f32<VE, NT>(mom, v, bn);
    gst<NT>(reinterpret_cast<u32x4*>(rep) + v, gpack<BF16>(tn));
  }
  if (do_tail) {
    float tn, bn;
    gnesterov(beta * static_cast<double>(dbar[tail]), theta[tail], mom[tail], lr, rho, tn, bn);
    theta[tail] = tn;
    mom[tail] = bn;
    gstore_scalar<BF16>(rep, tail, tn);
  }
}

template <typename Kern>
int gocc(Kern kernel, int threads) {
  int blocks = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, kernel, threads, 0) != hipSuccess || blocks < 1)
    blocks = 1;
  return blocks;
}

}  // namespace

// ------------------------------------------------------------ launchers

constexpr bool kGroupNT = true;  // every stream is touched once per pass

hipError_t launch_group_norm(bool bf16, int rows, const float* theta, const void* rep, float* delta,
                             int64_t n, double* partials, hipStream_t stream) {
  const int64_t nvec = n / (bf16 ? 8 : 4);
  if (bf16)
    hipLaunchKernelGGL((group_norm_kernel<true, kGroupNT>), dim3(rows), dim3(kGroupThreads), 0, stream, theta,
                       rep, delta, nvec, n, partials);
  else
    hipLaunchKernelGGL((group_norm_kernel<false, kGroupNT>), dim3(rows), dim3(kGroupThreads), 0, stream, theta,
                       rep, delta, nvec, n, partials);
  return hipGetLastError();
}

hipError_t launch_group_self(const double* partials, int rows, GroupRecord* rec, double* norm_out,
                             const GroupParams& prm, hipStream_t stream) {
  hipLaunchKernelGGL(group_self_kernel, dim3(1), dim3(kGroupOneBlock), 0, stream, partials, rows, rec, norm_out,
                     prm);
  return hipGetLastError();
}

hipError_t launch_group_weights(int blocks, const double* gathered, int K, int rank, GroupRecord* rec,
                                double* weight_out, float* delta, int64_t n, const GroupParams& prm,
                                hipStream_t stream) {
  hipLaunchKernelGGL(group_weights_kernel, dim3(blocks), dim3(kGroupThreads), 0, stream, gathered, K, rank, rec,
                     weight_out, delta, n, prm);
  return hipGetLastError();
}

hipError_t launch_group_dbar(int rows, const GroupRecord* rec, const float* dbar, int64_t n, double* partials,
                             hipStream_t stream) {
  hipLaunchKernelGGL((group_dbar_kernel<kGroupNT>), dim3(rows), dim3(kGroupThreads), 0, stream, rec, dbar, n,
                     partials);
  return hipGetLastError();
}

hipError_t launch_group_clip(const double* partials, int rows, GroupRecord* rec, const GroupParams& prm,
                             hipStream_t stream) {
  hipLaunchKernelGGL(group_clip_kernel, dim3(1), dim3(kGroupOneBlock), 0, stream, partials, rows, rec, prm);
  return hipGetLastError();
}

hipError_t launch_group_update(bool bf16, int blocks, const GroupRecord* rec, const float* dbar, float* theta,
                               float* mom, void* rep, int64_t n, double lr, double rho, hipStream_t stream) {
  const int64_t nvec = n / (bf16 ? 8 : 4);
  if (bf16)
    hipLaunchKernelGGL((group_update_kernel<true, kGroupNT>), dim3(blocks), dim3(kGroupUpdateThreads), 0, stream,
                       rec, dbar, theta, mom, rep, nvec, n, lr, rho);
  else
    hipLaunchKernelGGL((group_update_kernel<false, kGroupNT>), dim3(blocks), dim3(kGroupUpdateThreads), 0, stream,
                       rec, dbar, theta, mom, rep, nvec, n, lr, rho);
  return hipGetLastError();
}


int group_dbar_blocks_per_cu() { return gocc(group_dbar_kernel<kGroupNT>, kGroupThreads); }

}  // namespace edit
