// Device kernels of the EDiT outer synchronization step for gfx950.
//
// One step of one sync unit is three launches on one stream:
//
//   pass1  streams theta and the K replicas once and accumulates, per block,
//          the upper triangle of the Gram matrix  Gram_jk = <Delta_j, Delta_k>
//          of the pseudo gradients Delta_j = r_j - theta (Sec. 3.2).  The
//          diagonal gives the module norms G_j; the off-diagonal terms give
//          ||sum_j w_j Delta_j||^2 = w^T Gram w, so the clip factor of Eq. 4
//          is known before the update pass and the step needs two streaming
//          passes instead of three.
//   decide one block: fixed-order fp64 reduction of the per-block partials,
//          the EMA z-test and update (Eq. 1), rollback test, softmax weights
//          (Eq. 2), Gbar and beta (Eq. 4), per-worker coefficients beta*w_j.
//   pass2  streams theta, b and the replicas of the workers with a non-zero
//          coefficient, forms Delta_hat = sum_j beta w_j Delta_j (Eq. 3, 5),
//          applies Nesterov momentum and writes theta, b and all K replicas.
//
// Storage is fp32 (theta, b) and fp32/bf16 (replicas); arithmetic is fp64
// from the exact pseudo gradients on, rounded once when stored.
//
// The passes are HBM-bound (about 2-3 flop per byte at K = 8), so there is
// no MFMA: each lane moves 16-byte vectors (global_load_dwordx4), the grid is
// persistent (resident blocks only, grid-stride over 16-byte vectors) so the
// whole chip streams one contiguous window of every buffer at a time, and
// reductions go wave shuffle -> LDS -> per-block partial in a fixed order, so
// results are bitwise reproducible without atomics.
#include <type_traits>

#include "edit_outer_internal.h"

namespace edit {
namespace {

typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float float2_t __attribute__((ext_vector_type(2)));

template <int K>
struct ConstPtrs {
  const void* p[K];
};
template <int K>
struct MutPtrs {
  void* p[K];
};

template <bool BF16>
struct Vec {
  static constexpr int VE = BF16 ? 8 : 4;  // elements per 16-byte replica vector
};

// Element e of a 16-byte replica vector, widened to fp32 (exact).
template <bool BF16>
__device__ __forceinline__ float element(const uint4& raw, int e) {
  const uint32_t w[4] = {raw.x, raw.y, raw.z, raw.w};
  if constexpr (BF16) {
    const uint32_t word = w[e >> 1];
    return __uint_as_float((e & 1) ? (word & 0xffff0000u) : (word << 16));
  } else {
    return __uint_as_float(w[e]);
  }
}

template <bool BF16>
__device__ __forceinline__ float load_scalar(const void* base, int64_t i) {
  if constexpr (BF16) {
    const uint16_t h = reinterpret_cast<const uint16_t*>(base)[i];
    return __uint_as_float(static_cast<uint32_t>(h) << 16);
  } else {
    return reinterpret_cast<const float*>(base)[i];
  }
}

__device__ __forceinline__ uint32_t pack_bf16x2(float a, float b) {
  const float2_t f = {a, b};
  const bf16x2_t h = __builtin_convertvector(f, bf16x2_t);  // v_cvt_pk_bf16_f32, RNE
  return __builtin_bit_cast(uint32_t, h);
}

template <bool BF16>
__device__ __forceinline__ void store_scalar(void* base, int64_t i, float x) {
  if constexpr (BF16) {
    reinterpret_cast<uint16_t*>(base)[i] = static_cast<uint16_t>(pack_bf16x2(x, 0.f) & 0xffffu);
  } else {
    reinterpret_cast<float*>(base)[i] = x;
  }
}

// theta[v*VE .. v*VE+VE) as fp32.
template <int VE>
__device__ __forceinline__ void load_f32(const float* __restrict__ p, int64_t v, float (&x)[VE]) {
  const float4* q = reinterpret_cast<const float4*>(p) + v * (VE / 4);
#pragma unroll
  for (int h = 0; h < VE / 4; ++h) {
    const float4 t = q[h];
    x[4 * h + 0] = t.x;
    x[4 * h + 1] = t.y;
    x[4 * h + 2] = t.z;
    x[4 * h + 3] = t.w;
  }
}

template <int VE>
__device__ __forceinline__ void store_f32(float* __restrict__ p, int64_t v, const float (&x)[VE]) {
  float4* q = reinterpret_cast<float4*>(p) + v * (VE / 4);
#pragma unroll
  for (int h = 0; h < VE / 4; ++h) q[h] = make_float4(x[4 * h], x[4 * h + 1], x[4 * h + 2], x[4 * h + 3]);
}

// VE fp32 values -> one 16-byte replica vector.
template <bool BF16>
__device__ __forceinline__ uint4 pack(const float (&x)[Vec<BF16>::VE]) {
  if constexpr (BF16) {
    return make_uint4(pack_bf16x2(x[0], x[1]), pack_bf16x2(x[2], x[3]), pack_bf16x2(x[4], x[5]),
                      pack_bf16x2(x[6], x[7]));
  } else {
    return make_uint4(__float_as_uint(x[0]), __float_as_uint(x[1]), __float_as_uint(x[2]),
                      __float_as_uint(x[3]));
  }
}

// Sum over the 64 lanes of a wave, fixed butterfly order (same in every lane).
__device__ __forceinline__ double wave_sum(double x) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) x += __shfl_xor(x, m, 64);
  return x;
}

// ---------------------------------------------------------------- pass 1

// Element e of a 16-byte replica vector minus theta, in fp64: the pseudo
// gradient of that element, exact for every pair of fp32/bf16 inputs whose
// exponents differ by less than 29.
template <bool BF16>
__device__ __forceinline__ double delta64(const uint4& raw, int e, float th) {
  return static_cast<double>(element<BF16>(raw, e)) - static_cast<double>(th);
}

template <int K, bool BF16>
__global__ __launch_bounds__(kThreads) void pass1_gram_kernel(const float* __restrict__ theta,
                                                              ConstPtrs<K> reps, int64_t nvec,
                                                              int64_t n,
                                                              double* __restrict__ partials) {
  constexpr int NP = K * (K + 1) / 2;
  constexpr int VE = Vec<BF16>::VE;
  // fp64 products and sums: on CDNA3/4 a v_fma_f64 issues at the rate of an
  // unpacked v_fma_f32, so exactness costs no extra VALU cycles, and the
  // Gram identity for ||sum_j w_j Delta_j|| stays accurate even when the
  // workers' pseudo gradients nearly cancel.
  double acc[NP];
#pragma unroll
  for (int p = 0; p < NP; ++p) acc[p] = 0.0;

  const int64_t stride = static_cast<int64_t>(gridDim.x) * kThreads;
  for (int64_t v = static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x; v < nvec; v += stride) {
    float th[VE];
    load_f32<VE>(theta, v, th);
    uint4 raw[K];
#pragma unroll
    for (int j = 0; j < K; ++j) raw[j] = reinterpret_cast<const uint4*>(reps.p[j])[v];
#pragma unroll
    for (int e = 0; e < VE; ++e) {
      double d[K];
#pragma unroll
      for (int j = 0; j < K; ++j) d[j] = delta64<BF16>(raw[j], e, th[e]);
      int p = 0;
#pragma unroll
      for (int j = 0; j < K; ++j)
#pragma unroll
        for (int k = j; k < K; ++k, ++p) acc[p] = fma(d[j], d[k], acc[p]);
    }
  }

  // Ragged tail (fewer than VE elements past the last full vector): block 0.
  const int64_t i = nvec * VE + threadIdx.x;
  if (blockIdx.x == 0 && i < n) {
    double d[K];
    const double th = theta[i];
#pragma unroll
    for (int j = 0; j < K; ++j) d[j] = static_cast<double>(load_scalar<BF16>(reps.p[j], i)) - th;
    int p = 0;
#pragma unroll
    for (int j = 0; j < K; ++j)
#pragma unroll
      for (int k = j; k < K; ++k, ++p) acc[p] = fma(d[j], d[k], acc[p]);
  }

  // Block reduction: wave butterfly, then the four waves in order.
  __shared__ double red[kThreads / 64][NP];
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
#pragma unroll
  for (int p = 0; p < NP; ++p) {
    const double s = wave_sum(acc[p]);
    if (lane == 0) red[wave][p] = s;
  }
  __syncthreads();
  const int rows = gridDim.x;
  for (int p = threadIdx.x; p < NP; p += kThreads) {
    double s = red[0][p];
#pragma unroll
    for (int w = 1; w < kThreads / 64; ++w) s += red[w][p];
    partials[static_cast<int64_t>(p) * rows + blockIdx.x] = s;
  }
}

// ---------------------------------------------------------------- decide

__device__ __forceinline__ int pair_index(int K, int j, int k) {  // j <= k
  return j * K - (j * (j - 1)) / 2 + (k - j);
}

template <int K>
__global__ __launch_bounds__(kThreads) void decide_kernel(const double* __restrict__ partials,
                                                          int rows, UnitRecord* __restrict__ rec,
                                                          DecideParams prm) {
  constexpr int NP = K * (K + 1) / 2;
  __shared__ double gram[NP];
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  for (int p = wave; p < NP; p += kThreads / 64) {
    double s = 0.0;
    for (int r = lane; r < rows; r += 64) s += partials[static_cast<int64_t>(p) * rows + r];
    s = wave_sum(s);
    if (lane == 0) gram[p] = s;
  }
  __syncthreads();
  if (threadIdx.x != 0) return;

  const bool ae = prm.flags & EDIT_AE;
  const bool wa = prm.flags & EDIT_WA;
  const bool gc = prm.flags & EDIT_GC;
  const int64_t t = rec->round;
  const bool z_test = ae && t >= prm.warmup;

  // Norms and anomaly elimination (Sec. 3.2): the z-test z = (G - mu)/sigma > delta
  // is taken as G - mu > delta*sigma against the state before this round;
  // a non-finite norm is always flagged.
  double G[K];
  bool bad[K];
  int n_ok = 0;
#pragma unroll
  for (int j = 0; j < K; ++j) {
    G[j] = sqrt(gram[pair_index(K, j, j)]);
    bool flag = !isfinite(G[j]);
    if (z_test && !flag) flag = (G[j] - rec->mu[j]) > prm.delta * rec->sigma[j];
    bad[j] = flag;
    n_ok += flag ? 0 : 1;
    rec->norm[j] = G[j];
    rec->anomalous[j] = flag ? 1 : 0;
  }
  // Eq. 1 for the workers that were not flagged.
  if (ae) {
#pragma unroll
    for (int j = 0; j < K; ++j) {
      if (bad[j]) continue;
      const double mu = prm.alpha * G[j] + (1.0 - prm.alpha) * rec->mu[j];
      const double dev = G[j] - mu;
      const double sg = rec->sigma[j];
      rec->sigma[j] = sqrt((1.0 - prm.alpha) * sg * sg + prm.alpha * dev * dev);
      rec->mu[j] = mu;
    }
  }

  double w[K];
  double gbar = 0.0, beta = 0.0;
  if (n_ok == 0) {
#pragma unroll
    for (int j = 0; j < K; ++j) w[j] = 0.0;
  } else {
    if (wa) {  // Eq. 2 as a softmax of -G over the unflagged workers, shifted by min G
      double g0 = INFINITY;
#pragma unroll
      for (int j = 0; j < K; ++j)
        if (!bad[j] && G[j] < g0) g0 = G[j];
      double gamma = 0.0;
#pragma unroll
      for (int j = 0; j < K; ++j) {
        w[j] = bad[j] ? 0.0 : exp(-(G[j] - g0));
        gamma += w[j];
      }
#pragma unroll
      for (int j = 0; j < K; ++j) w[j] /= gamma;
    } else {
#pragma unroll
      for (int j = 0; j < K; ++j) w[j] = bad[j] ? 0.0 : 1.0 / n_ok;
    }
    // ||sum_j w_j Delta_j||^2 = sum_jk w_j w_k Gram_jk (Eq. 3-4).
    double q = 0.0;
#pragma unroll
    for (int j = 0; j < K; ++j) {
      if (bad[j]) continue;
#pragma unroll
      for (int k = 0; k < K; ++k) {
        if (bad[k]) continue;
        const double g = j <= k ? gram[pair_index(K, j, k)] : gram[pair_index(K, k, j)];
        q += w[j] * w[k] * g;
      }
    }
    gbar = sqrt(fmax(q, 0.0));
    beta = gc ? fmin(prm.phi / (gbar + prm.eps), 1.0) : 1.0;
  }

  int first = -1;
#pragma unroll
  for (int j = 0; j < K; ++j) {
    const double c = beta * w[j];
    rec->weight[j] = w[j];
    rec->coef[j] = c;
    if (c != 0.0 && first < 0) first = j;
  }
  // The update pass loads slot j from worker src[j]: itself when it
  // contributes, otherwise a contributing worker (a cache hit, and never the
  // data of a flagged worker, which may hold NaN).
#pragma unroll
  for (int j = 0; j < K; ++j) rec->src[j] = (rec->coef[j] != 0.0 || first < 0) ? j : first;
  rec->use_deltas = first >= 0 ? 1 : 0;
  rec->rollback = n_ok == 0 ? 1 : 0;
  rec->synced_norm = gbar;
  rec->clip_coef = beta;
  rec->z_tested = z_test ? 1 : 0;
  rec->stepped = 1;
  rec->round = t + 1;
}

// ---------------------------------------------------------------- pass 2

// theta' and b' of one element, in fp64 from fp32 inputs (rounded once on store):
//   Delta_hat = sum_j c_j (r_j - theta), c_j = beta w_j      (Eq. 3, 5)
//   g = -Delta_hat;  b' = rho b + g;  theta' = theta - nu (g + rho b')
__device__ __forceinline__ void nesterov(double dhat, float th, float b, double lr, double rho,
                                         float& th_out, float& b_out) {
  const double g = -dhat;
  const double bn = fma(rho, static_cast<double>(b), g);
  th_out = static_cast<float>(static_cast<double>(th) - lr * fma(rho, bn, g));
  b_out = static_cast<float>(bn);
}

template <int K, bool BF16>
__global__ __launch_bounds__(kThreads) void pass2_update_kernel(float* __restrict__ theta,
                                                                float* __restrict__ mom,
                                                                MutPtrs<K> reps,
                                                                const UnitRecord* __restrict__ rec,
                                                                int64_t nvec, int64_t n, double lr,
                                                                double rho) {
  constexpr int VE = Vec<BF16>::VE;
  const int64_t stride = static_cast<int64_t>(gridDim.x) * kThreads;
  const int64_t v0 = static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x;
  const int64_t tail = nvec * VE + threadIdx.x;
  const bool do_tail = blockIdx.x == 0 && tail < n;

  if (rec->rollback) {  // every worker flagged: replicas <- theta_t, nothing else moves
    for (int64_t v = v0; v < nvec; v += stride) {
      float th[VE];
      load_f32<VE>(theta, v, th);
      const uint4 out = pack<BF16>(th);
#pragma unroll
      for (int j = 0; j < K; ++j) reinterpret_cast<uint4*>(reps.p[j])[v] = out;
    }
    if (do_tail) {
      const float th = theta[tail];
#pragma unroll
      for (int j = 0; j < K; ++j) store_scalar<BF16>(reps.p[j], tail, th);
    }
    return;
  }

  double c[K];
  const uint4* src[K];
#pragma unroll
  for (int j = 0; j < K; ++j) {
    c[j] = rec->coef[j];
    const int s = rec->src[j];
    const void* ptr = reps.p[0];
#pragma unroll
    for (int i = 1; i < K; ++i) ptr = (s == i) ? reps.p[i] : ptr;
    src[j] = reinterpret_cast<const uint4*>(ptr);
  }
  const bool use = rec->use_deltas;

  for (int64_t v = v0; v < nvec; v += stride) {
    float th[VE], b[VE];
    double acc[VE];
    load_f32<VE>(theta, v, th);
    load_f32<VE>(mom, v, b);
#pragma unroll
    for (int e = 0; e < VE; ++e) acc[e] = 0.0;
    if (use) {
      uint4 raw[K];
#pragma unroll
      for (int j = 0; j < K; ++j) raw[j] = src[j][v];
#pragma unroll
      for (int j = 0; j < K; ++j)
#pragma unroll
        for (int e = 0; e < VE; ++e) acc[e] = fma(c[j], delta64<BF16>(raw[j], e, th[e]), acc[e]);
    }
    float tn[VE], bn[VE];
#pragma unroll
    for (int e = 0; e < VE; ++e) nesterov(acc[e], th[e], b[e], lr, rho, tn[e], bn[e]);
    store_f32<VE>(theta, v, tn);
    store_f32<VE>(mom, v, bn);
    const uint4 out = pack<BF16>(tn);
#pragma unroll
    for (int j = 0; j < K; ++j) reinterpret_cast<uint4*>(reps.p[j])[v] = out;
  }

  if (do_tail) {
    const float th = theta[tail];
    double acc = 0.0;
    if (use) {
#pragma unroll
      for (int j = 0; j < K; ++j)
        acc = fma(c[j],
                  static_cast<double>(load_scalar<BF16>(reinterpret_cast<const void*>(src[j]), tail)) -
                      static_cast<double>(th),
                  acc);
    }
    float tn, bn;
    nesterov(acc, th, mom[tail], lr, rho, tn, bn);
    theta[tail] = tn;
    mom[tail] = bn;
#pragma unroll
    for (int j = 0; j < K; ++j) store_scalar<BF16>(reps.p[j], tail, tn);
  }
}

// ------------------------------------------------------------ copy probe

__global__ __launch_bounds__(kThreads) void copy_kernel(uint4* __restrict__ dst,
                                                       const uint4* __restrict__ src,
                                                       int64_t nvec) {
  const int64_t stride = static_cast<int64_t>(gridDim.x) * kThreads;
  for (int64_t v = static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x; v < nvec; v += stride)
    dst[v] = src[v];
}

// ------------------------------------------------------------ launchers

template <int K, bool BF16>
hipError_t pass1_launch(int blocks, const float* theta, const void* const* reps, int64_t n,
                        double* partials, hipStream_t stream) {
  ConstPtrs<K> rp;
  for (int j = 0; j < K; ++j) rp.p[j] = reps[j];
  const int64_t nvec = n / Vec<BF16>::VE;
  hipLaunchKernelGGL((pass1_gram_kernel<K, BF16>), dim3(blocks), dim3(kThreads), 0, stream, theta,
                     rp, nvec, n, partials);
  return hipGetLastError();
}

template <int K, bool BF16>
hipError_t pass2_launch(int blocks, float* theta, float* mom, void* const* reps,
                        const UnitRecord* rec, int64_t n, double lr, double rho, hipStream_t stream) {
  MutPtrs<K> rp;
  for (int j = 0; j < K; ++j) rp.p[j] = reps[j];
  const int64_t nvec = n / Vec<BF16>::VE;
  hipLaunchKernelGGL((pass2_update_kernel<K, BF16>), dim3(blocks), dim3(kThreads), 0, stream, theta,
                     mom, rp, rec, nvec, n, lr, rho);
  return hipGetLastError();
}

template <int K>
hipError_t decide_launch(const double* partials, int rows, UnitRecord* rec, const DecideParams& prm,
                         hipStream_t stream) {
  hipLaunchKernelGGL((decide_kernel<K>), dim3(1), dim3(kThreads), 0, stream, partials, rows, rec, prm);
  return hipGetLastError();
}

template <typename Kern>
int occupancy(Kern kernel) {
  int blocks = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, kernel, kThreads, 0) != hipSuccess ||
      blocks < 1)
    blocks = 1;
  return blocks;
}

}  // namespace

#define EDIT_FOR_EACH_K(X) \
  X(1) X(2) X(3) X(4) X(5) X(6) X(7) X(8) X(9) X(10) X(11) X(12) X(13) X(14) X(15) X(16)

hipError_t launch_pass1(int K, bool bf16, int blocks, const float* theta, const void* const* reps,
                        int64_t n, double* partials, hipStream_t stream) {
  switch (K) {
#define EDIT_CASE(KK)                                                                        \
  case KK:                                                                                   \
    return bf16 ? pass1_launch<KK, true>(blocks, theta, reps, n, partials, stream)           \
                : pass1_launch<KK, false>(blocks, theta, reps, n, partials, stream);
    EDIT_FOR_EACH_K(EDIT_CASE)
#undef EDIT_CASE
    default:
      return hipErrorInvalidValue;
  }
}

hipError_t launch_decide(int K, const double* partials, int rows, UnitRecord* rec,
                         const DecideParams& prm, hipStream_t stream) {
  switch (K) {
#define EDIT_CASE(KK) \
  case KK:            \
    return decide_launch<KK>(partials, rows, rec, prm, stream);
    EDIT_FOR_EACH_K(EDIT_CASE)
#undef EDIT_CASE
    default:
      return hipErrorInvalidValue;
  }
}

hipError_t launch_pass2(int K, bool bf16, int blocks, float* theta, float* mom, void* const* reps,
                        const UnitRecord* rec, int64_t n, double lr, double rho, hipStream_t stream) {
  switch (K) {
#define EDIT_CASE(KK)                                                                          \
  case KK:                                                                                     \
    return bf16 ? pass2_launch<KK, true>(blocks, theta, mom, reps, rec, n, lr, rho, stream)    \
                : pass2_launch<KK, false>(blocks, theta, mom, reps, rec, n, lr, rho, stream);
    EDIT_FOR_EACH_K(EDIT_CASE)
#undef EDIT_CASE
    default:
      return hipErrorInvalidValue;
  }
}

hipError_t launch_copy(void* dst, const void* src, int64_t nbytes, int blocks, hipStream_t stream) {
  hipLaunchKernelGGL(copy_kernel, dim3(blocks), dim3(kThreads), 0, stream,
                     reinterpret_cast<uint4*>(dst), reinterpret_cast<const uint4*>(src), nbytes / 16);
  return hipGetLastError();
}

int pass1_blocks_per_cu(int K, bool bf16) {
  switch (K) {
#define EDIT_CASE(KK) \
  case KK:            \
    return bf16 ? occupancy(pass1_gram_kernel<KK, true>) : occupancy(pass1_gram_kernel<KK, false>);
    EDIT_FOR_EACH_K(EDIT_CASE)
#undef EDIT_CASE
    default:
      return 1;
  }
}

int pass2_blocks_per_cu(int K, bool bf16) {
  switch (K) {
#define EDIT_CASE(KK) \
  case KK:            \
    return bf16 ? occupancy(pass2_update_kernel<KK, true>) : occupancy(pass2_update_kernel<KK, false>);
    EDIT_FOR_EACH_K(EDIT_CASE)
#undef EDIT_CASE
    default:
      return 1;
  }
}

}  // namespace edit
