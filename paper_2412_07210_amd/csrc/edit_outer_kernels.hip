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
//   decide one block: fixed-order reduction of the per-block partials, then
//          one wave (worker j in lane j) takes the decision: EMA z-test and
//          update (Eq. 1), rollback test, softmax weights (Eq. 2), Gbar and
//          beta (Eq. 4), coefficients beta*w_j.
//   pass2  streams theta, b and the replicas of the workers with a non-zero
//          coefficient, forms Delta_hat = sum_j beta w_j Delta_j (Eq. 3, 5),
//          applies Nesterov momentum and writes theta, b and all K replicas.
//
// Storage is fp32 (theta, b) and fp32/bf16 (replicas); arithmetic is fp64
// from the exact pseudo gradients on, rounded once when stored.
//
// The passes are HBM-bound (2-4 flop per byte at K = 8).  Lanes move 16-byte
// vectors (global_load_dwordx4).  Pass 1 runs a persistent grid of one block
// per CU holding all the waves the CU runs of it (grid-stride), so the chip
// streams one contiguous window of every buffer at a time and the decision
// reduces one partial row per CU; up to K = 8 each lane double-buffers its
// vectors (the loads of trip t+1 are in flight while trip t is computed), so
// the fp64 work hides under the memory latency even at 2 waves per SIMD.
// Above K = 8 the Gram is a rank-n update on the fp64 matrix cores
// (v_mfma_f64_4x4x4f64 tiles), which the VALU could not hold in registers.
// Pass 2, which writes as much as it reads, instead gives each thread one
// vector and lets the block dispatcher order the traffic (see there).
//
// Also here: the Gram pass of two units of a round in one launch
// (pass1_gram_pair_kernel), the small launch of a round that steps units of
// one Gram-pass block whole (round_small_kernel; the bodies of pass 1 and
// pass 2 are the fragments gram_rows_valu.inc, gram_rows_mfma.inc and
// update_vector_at.inc, shared with the kernels above), the Gram
// export/import of a sharded module
// (gram_reduce_kernel, decide_gram_kernel), the one-pass mean step used when
// no penalty component is on (fused_mean_kernel, fused_finish_kernel), and a
// plain copy kernel for bandwidth and counter calibration.  Reductions go
// wave shuffle -> LDS -> per-block partial -> one block in a fixed order, so
// results are bitwise reproducible.
#include "edit_outer_internal.h"

#include <algorithm>

// Compiled once per range of worker counts (EDIT_K_RANGES); the build passes
// the range's first and last K.
#if !defined(EDIT_K_FIRST) || !defined(EDIT_K_LAST)
#error "compile with -DEDIT_K_FIRST=<first K> -DEDIT_K_LAST=<last K> of one of EDIT_K_RANGES"
#endif

namespace edit {
namespace {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
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

// 16-byte global accesses; NT marks them non-temporal (streaming) in the cache.
template <bool NT, typename T>
__device__ __forceinline__ T ld16(const T* p) {
  if constexpr (NT)
    return __builtin_nontemporal_load(p);
  else
    return *p;
}
template <bool NT, typename T>
__device__ __forceinline__ void st16(T* p, T v) {
  if constexpr (NT)
    __builtin_nontemporal_store(v, p);
  else
    *p = v;
}

// Element e of a 16-byte replica vector, widened to fp32 (exact).
template <bool BF16>
__device__ __forceinline__ float element(const u32x4& raw, int e) {
  if constexpr (BF16) {
    const uint32_t word = raw[e >> 1];
    return __uint_as_float((e & 1) ? (word & 0xffff0000u) : (word << 16));
  } else {
    return __uint_as_float(raw[e]);
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

// fp32 values [v*VE, v*VE+VE) of a theta/momentum buffer.
template <int VE, bool NT>
__device__ __forceinline__ void load_f32(const float* p, int64_t v, float (&x)[VE]) {
  const f32x4* q = reinterpret_cast<const f32x4*>(p) + v * (VE / 4);
#pragma unroll
  for (int h = 0; h < VE / 4; ++h) {
    const f32x4 t = ld16<NT>(q + h);
#pragma unroll
    for (int c = 0; c < 4; ++c) x[4 * h + c] = t[c];
  }
}

template <int VE, bool NT>
__device__ __forceinline__ void store_f32(float* p, int64_t v, const float (&x)[VE]) {
  f32x4* q = reinterpret_cast<f32x4*>(p) + v * (VE / 4);
#pragma unroll
  for (int h = 0; h < VE / 4; ++h) {
    f32x4 t;
#pragma unroll
    for (int c = 0; c < 4; ++c) t[c] = x[4 * h + c];
    st16<NT>(q + h, t);
  }
}

// VE fp32 values -> one 16-byte replica vector.
template <bool BF16>
__device__ __forceinline__ u32x4 pack(const float (&x)[Vec<BF16>::VE]) {
  u32x4 r;
  if constexpr (BF16) {
#pragma unroll
    for (int c = 0; c < 4; ++c) r[c] = pack_bf16x2(x[2 * c], x[2 * c + 1]);
  } else {
#pragma unroll
    for (int c = 0; c < 4; ++c) r[c] = __float_as_uint(x[c]);
  }
  return r;
}

// Element e of a replica vector minus theta, in fp64: the pseudo gradient of
// that element, exact for fp32/bf16 inputs whose exponents differ by < 29.
template <bool BF16>
__device__ __forceinline__ double delta64(const u32x4& raw, int e, float th) {
  return static_cast<double>(element<BF16>(raw, e)) - static_cast<double>(th);
}

// A field of a unit record read by the update pass.  When the record was
// written earlier in the same launch (the single-block path, kFresh), the
// load is a relaxed atomic at work-group scope: always a vector memory
// instruction, which sees the other waves' stores once a barrier has
// ordered them, whereas a scalar-cache load could return stale data.  A
// record written by an earlier launch is read with a plain load.
template <bool kFresh, typename T>
__device__ __forceinline__ T rec_load(const T* p) {
  if constexpr (kFresh)
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
  else
    return *p;
}

// Sum over the 64 lanes of a wave, fixed butterfly order (same in every lane).
__device__ __forceinline__ double wave_sum(double x) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) x += __shfl_xor(x, m, 64);
  return x;
}

__device__ __forceinline__ int pair_index(int K, int j, int k) {  // j <= k
  return j * K - (j * (j - 1)) / 2 + (k - j);
}

// ------------------------------------------------------------- decision

constexpr int kDecideThreads = 1024;  // one block; wide so the partial loads overlap
constexpr int kReduceLogical = 1024;  // logical threads of the partial reduction

// Reduce the per-block Gram partials [NP][rows] in a fixed order into
// gram[NP] (shared memory).  Logical thread lt takes pair lt / T and rows
// lt % T, lt % T + T, ... (T phases per pair, at most 64), with 16 loads in
// flight, and the T phase sums of a pair are then added in phase order.
// The partials were just written by every XCD's blocks, so the loads come
// from the Infinity Cache or HBM and the reduction is latency-bound: many
// independent loads per thread matter more than anything else here.  The
// order depends on neither the block size nor the unrolling, so a standalone
// decision kernel, one folded into a pass-1 launch and the Gram export agree
// bit for bit.  `scratch` holds kReduceLogical doubles of shared memory.
template <int K, int kBlockThreads>
__device__ void reduce_partials(const double* partials, int rows, double* gram, double* scratch) {
  constexpr int NP = K * (K + 1) / 2;
  constexpr int T = kReduceLogical / NP < 64 ? kReduceLogical / NP : 64;
  for (int lt = threadIdx.x; lt < NP * T; lt += kBlockThreads) {
    const int p = lt / T, ph = lt % T;
    const double* src = partials + static_cast<int64_t>(p) * rows;
    double acc = 0.0;
#pragma unroll 16
    for (int r = ph; r < rows; r += T) acc += __builtin_nontemporal_load(src + r);
    scratch[lt] = acc;
  }
  __syncthreads();
  for (int p = threadIdx.x; p < NP; p += kBlockThreads) {
    double g = 0.0;
    for (int ph = 0; ph < T; ++ph) g += scratch[p * T + ph];
    gram[p] = g;
  }
}

// The state a decision starts from: round counter and each worker's EMA
// pair, loaded by the deciding wave before the partial reduction so that
// their latency hides behind it.
struct DecideState {
  int64_t round;
  double mu, sigma;  // of the lane's worker (lane < K)
};

template <int K>
__device__ __forceinline__ DecideState load_decide_state(const UnitRecord* rec) {
  const int lane = threadIdx.x & 63;
  DecideState st{rec->round, 0.0, 0.0};
  if (lane < K) {
    st.mu = rec->mu[lane];
    st.sigma = rec->sigma[lane];
  }
  return st;
}

// The decision of one step from the unit's Gram matrix, taken by one wave:
// worker j's norm, z-test, EMA update and softmax term live in lane j; the
// cross-lane steps (min, sums, first contributing worker) are fixed-order
// butterflies and ballots, so the result is reproducible bit for bit.
template <int K>
__device__ void decide(const double* gram, UnitRecord* rec, const DecideParams& prm,
                       const DecideState& st) {
  const int lane = threadIdx.x & 63;
  const bool ae = prm.flags & EDIT_AE;
  const bool wa = prm.flags & EDIT_WA;
  const bool gc = prm.flags & EDIT_GC;
  const int64_t t = st.round;
  const bool z_test = ae && t >= prm.warmup;
  const bool mine = lane < K;

  // Norms and anomaly elimination (Sec. 3.2): the z-test z = (G - mu)/sigma > delta
  // is taken as G - mu > delta*sigma against the state before this round; a
  // non-finite norm is always flagged.  Eq. 1 then updates the unflagged.
  double G = 0.0;
  bool bad = true;
  if (mine) {
    G = sqrt(gram[pair_index(K, lane, lane)]);
    bad = !isfinite(G);
    const double mu0 = st.mu;
    const double sg0 = st.sigma;
    if (z_test && !bad) bad = (G - mu0) > prm.delta * sg0;
    rec->norm[lane] = G;
    rec->anomalous[lane] = bad ? 1 : 0;
    if (ae && !bad) {
      const double mu = prm.alpha * G + (1.0 - prm.alpha) * mu0;
      const double dev = G - mu;
      rec->sigma[lane] = sqrt((1.0 - prm.alpha) * sg0 * sg0 + prm.alpha * dev * dev);
      rec->mu[lane] = mu;
    }
  }
  const bool ok = mine && !bad;
  const int n_ok = __popcll(__ballot(ok));

  double w = 0.0, gbar = 0.0, beta = 0.0;
  if (n_ok > 0) {
    if (wa) {  // Eq. 2 as a softmax of -G over the unflagged workers, shifted by min G
      double g0 = ok ? G : INFINITY;
#pragma unroll
      for (int m = 32; m >= 1; m >>= 1) g0 = fmin(g0, __shfl_xor(g0, m, 64));
      const double e = ok ? exp(-(G - g0)) : 0.0;
      w = e / wave_sum(e);
    } else {
      w = ok ? 1.0 / n_ok : 0.0;
    }
    // ||sum_j w_j Delta_j||^2 = sum_jk w_j w_k Gram_jk (Eq. 3-4); every lane
    // takes part in every shuffle (uniform trip count).
    double q = 0.0;
#pragma unroll
    for (int it = 0; it < (K * K + 63) / 64; ++it) {
      const int pk = lane + 64 * it;
      const int pkc = pk < K * K ? pk : 0;
      const int j = pkc / K, k = pkc % K;
      const double wj = __shfl(w, j, 64);
      const double wk = __shfl(w, k, 64);
      const double g = j <= k ? gram[pair_index(K, j, k)] : gram[pair_index(K, k, j)];
      // flagged workers have w = 0 and may have non-finite Gram entries
      if (pk < K * K && wj != 0.0 && wk != 0.0) q += wj * wk * g;
    }
    gbar = sqrt(fmax(wave_sum(q), 0.0));
    beta = gc ? fmin(prm.phi / (gbar + prm.eps), 1.0) : 1.0;
  }

  // The update pass loads slot j from worker src[j]: itself when it
  // contributes, otherwise a contributing worker (a cache hit, and never the
  // data of a flagged worker, which may hold NaN).
  const double c = beta * w;
  const unsigned long long nz = __ballot(mine && c != 0.0);
  const int first = nz ? __ffsll(static_cast<long long>(nz)) - 1 : -1;
  if (mine) {
    rec->weight[lane] = w;
    rec->coef[lane] = c;
    rec->src[lane] = (c != 0.0 || first < 0) ? lane : first;
  }
  if (lane == 0) {
    rec->use_deltas = first >= 0 ? 1 : 0;
    rec->rollback = n_ok == 0 ? 1 : 0;
    rec->synced_norm = gbar;
    rec->clip_coef = beta;
    rec->z_tested = z_test ? 1 : 0;
    rec->stepped = 1;
    rec->round = t + 1;
  }
}

// ---------------------------------------------------------------- pass 1

// The decision of the previous unit of a round, taken by block 0 of a pass-1
// launch (partials == nullptr: none).  The previous unit's pass 1 finished
// before this launch began, so its partials are visible, and its decision
// costs no serial time of its own.
struct PrevDecide {
  const double* partials;
  int rows;
  UnitRecord* rec;
};

// Threads per block of the Gram pass.  The MFMA version runs one block per
// CU holding all its resident waves (3 per SIMD up to K = 16, 2 above, where
// the 21 to 36 accumulator tiles and the double-buffered vectors of eight
// worker groups need up to 256 VGPRs per lane), so the block reduction
// combines them and the decision reduces one partial row per CU: at K = 16
// that row count (255 against 767) took the decision from 26 to 12 us.  The
// VALU version keeps 256-thread blocks: one 512-thread block per CU shortened
// its decision too, but made the whole 1B step 0.7% slower (same-box A/B).
template <int K>
constexpr int pass1_threads() {
  return K <= 8 ? 256 : (K <= 16 ? 768 : 512);
}

template <int K, int kBlockThreads>
__device__ void run_prev_decide(const PrevDecide& prev, const DecideParams& prm) {
  __shared__ double gram[K * (K + 1) / 2];
  __shared__ double scratch[kReduceLogical];
  const DecideState st = load_decide_state<K>(prev.rec);
  reduce_partials<K, kBlockThreads>(prev.partials, prev.rows, gram, scratch);
  __syncthreads();
  if (threadIdx.x < 64) decide<K>(gram, prev.rec, prm, st);
}


// Gram contributions of one 16-byte vector of every replica.
template <int K, bool BF16>
__device__ __forceinline__ void gram_vector(double (&acc)[K * (K + 1) / 2], const u32x4 (&raw)[K],
                                            const float (&th)[Vec<BF16>::VE]) {
#pragma unroll
  for (int e = 0; e < Vec<BF16>::VE; ++e) {
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

// theta and every replica at vector v (< nvec).  Unguarded: the caller
// clamps v, so that no load sits under a lane mask; a masked load makes the
// compiler wait for the next trip's loads before computing this one.
template <int K, bool BF16, bool NT>
__device__ __forceinline__ void load_pass1(const float* theta, const ConstPtrs<K>& reps, int64_t v,
                                           float (&th)[Vec<BF16>::VE], u32x4 (&raw)[K]) {
  load_f32<Vec<BF16>::VE, NT>(theta, v, th);
#pragma unroll
  for (int j = 0; j < K; ++j) raw[j] = ld16<NT>(reinterpret_cast<const u32x4*>(reps.p[j]) + v);
}

template <int K, bool BF16, bool NT>
__global__ __launch_bounds__(pass1_threads<K>()) void pass1_gram_kernel(const float* __restrict__ theta,
                                                              ConstPtrs<K> reps, int64_t nvec,
                                                              int64_t n,
                                                              double* __restrict__ partials,
                                                              PrevDecide prev, DecideParams prm) {
  constexpr int NP = K * (K + 1) / 2;
  constexpr int VE = Vec<BF16>::VE;
  const int first = prev.partials ? 1 : 0;  // block 0 may take the previous unit's decision
  if (first && blockIdx.x == 0) {
    run_prev_decide<K, pass1_threads<K>()>(prev, prm);
    return;
  }
  const int b = static_cast<int>(blockIdx.x) - first;  // this block's partial row
  const int rows = static_cast<int>(gridDim.x) - first;
#include "gram_rows_valu.inc"
}

// The decisions of up to two earlier units of a round (prev1 only with
// prev0), one after the other in the calling block.
template <int K>
__device__ void run_prev_decisions(const PrevDecide& prev0, const PrevDecide& prev1,
                                   const DecideParams& prm) {
  run_prev_decide<K, pass1_threads<K>()>(prev0, prm);
  if (prev1.partials) {
    __syncthreads();  // the first decision has read the shared Gram
    run_prev_decide<K, pass1_threads<K>()>(prev1, prm);
  }
}

// One unit of a two-unit Gram launch (rows == 0: none).
template <int K>
struct Pass1Part {
  const float* theta;
  ConstPtrs<K> reps;
  int64_t nvec;
  int64_t n;
  double* partials;
  int rows;
};

// Pass 1 of two consecutive units of a round in one launch (K <= 8).  Each
// block writes its partial row of the first unit, then the same row of the
// second, so each unit gets exactly the partials of its own launch (same
// rows, same order).  The persistent grid then starts and drains once for
// the two units instead of twice; that start and drain costs about 13 us
// per launch whatever the unit size.  Block 0 may take the decisions of the
// two units before them.  UNITS = 1 is the launch of one unit that takes
// two such decisions.
template <int K, bool BF16, bool NT, int UNITS>
__global__ __launch_bounds__(pass1_threads<K>()) void pass1_gram_pair_kernel(Pass1Part<K> unit0,
                                                                   Pass1Part<K> unit1,
                                                                   PrevDecide prev0,
                                                                   PrevDecide prev1,
                                                                   DecideParams prm) {
  constexpr int NP = K * (K + 1) / 2;
  constexpr int VE = Vec<BF16>::VE;
  const int first = prev0.partials ? 1 : 0;
  if (first && blockIdx.x == 0) {
    run_prev_decisions<K>(prev0, prev1, prm);
    return;
  }
  const int b = static_cast<int>(blockIdx.x) - first;  // this block's partial row of each unit
#pragma unroll 1
  for (int w = 0; w < UNITS; ++w) {
    const int rows = w == 0 ? unit0.rows : unit1.rows;
    if (b >= rows) continue;
    if (w == 1) __syncthreads();  // the first unit's block reduction has read red[]
    const float* __restrict__ theta = w == 0 ? unit0.theta : unit1.theta;
    ConstPtrs<K> reps;
#pragma unroll
    for (int j = 0; j < K; ++j) reps.p[j] = w == 0 ? unit0.reps.p[j] : unit1.reps.p[j];
    const int64_t nvec = w == 0 ? unit0.nvec : unit1.nvec;
    const int64_t n = w == 0 ? unit0.n : unit1.n;
    double* __restrict__ partials = w == 0 ? unit0.partials : unit1.partials;
#include "gram_rows_valu.inc"
  }
}

// Pass 1 for 8 < K <= 32: the Gram matrix sum_i d_i d_i^T over the unit's
// elements is a rank-n update, and with K(K+1)/2 = 136 to 528 fp64 sums per
// lane a VALU version runs out of registers.  It runs on the fp64 matrix
// cores as v_mfma_f64_4x4x4f64, four independent 4x4x4 products per wave
// instruction (blocks b = 0..3).  The workers form G = ceil(K/4) groups of
// four and the Gram matrix 4x4 tiles (I, J); only the G(G+1)/2 tiles with
// I <= J are formed (10 of 16 at K = 16, 36 of 64 at K = 32): 160 products
// per element at K = 16 where the 16x16x4 instruction forms all 256, and
// this one also sustains a higher share of the fp64 matrix peak.  On gfx950 the fp64 matrix work and the fp64
// vector work of the deltas (widening, subtracting theta) do not overlap,
// so the pass is bound by their sum rather than by HBM.
//
// Operand layout of the instruction on gfx950 (checked with a one-hot
// probe): lane l holds A[i][k] and B[k][j] of block b with i = j = l % 4,
// b = (l / 4) % 4, k = l / 16, and the result D[i][j] of block b sits in
// lane j + 4b + 16i.  So the four lanes of a quad q = l / 4 share (b, k):
// they take one element, lane c = l % 4 holding the pseudo gradients of
// workers c, c+4, c+8, c+12 of it, and for tile (I, J) a lane passes its
// group-I value as A and its group-J value as B.  Each instruction adds the
// products of 16 elements (one per quad) into the tile, block b summing the
// quads b, b+4, b+8, b+12; the blocks are added at the end.

// Vector slots per lane per loop trip of the matrix-core pass (two, or
// loads two trips ahead, measured no faster and need 512-thread blocks).
constexpr int kMfmaSlots = 1;
// Load buffers per lane in the matrix-core pass's loop: two (the next trip's
// loads in flight while one is computed).  With every load unmasked, three
// buffers and 1024-thread blocks measured within 1% of this at K = 16 (A/B
// on one box): the pass is not waiting on memory latency.  Its matrix-core
// and vector instructions share one issue port and take its time.
template <int K>
constexpr int kMfmaDepth() {
  return 2;
}

template <int K>
struct Tiles4 {
  static constexpr int G = (K + 3) / 4;      // worker groups of four
  static constexpr int T = G * (G + 1) / 2;  // tiles (I, J), I <= J
};

// One vector slot of a quad: the whole theta vector (every lane of the quad
// loads it; the L1 serves the repeats, which measured faster than loading a
// quarter per lane and broadcasting it by DPP moves, eight more vector
// instructions per slot) and lane c's groups' replica vectors.
template <int G, bool BF16>
struct Quad4 {
  static constexpr int TH = Vec<BF16>::VE;
  u32x4 raw[G];
  float th[TH];
};

// Vector v (< nvec) of theta and of this lane's replicas (rep[g] is worker
// 4g + lane % 4).  Lanes of workers >= K (act false, only in the last group
// when K is not a multiple of 4) feed zeros.  No bounds guard: the caller
// clamps v, so that no load sits under a lane mask and the loads of later
// trips stay in flight.
template <int G, bool BF16, bool NT>
__device__ __forceinline__ void load_quad4(const float* theta, const void* const (&rep)[G],
                                           const bool (&act)[G], int64_t v, Quad4<G, BF16>& q) {
  load_f32<Vec<BF16>::VE, NT>(theta, v, q.th);
#pragma unroll
  for (int g = 0; g < G; ++g)
    q.raw[g] = act[g] ? ld16<NT>(reinterpret_cast<const u32x4*>(rep[g]) + v) : u32x4{0u, 0u, 0u, 0u};
}

// A quad whose vector lies past the unit's end contributes nothing.
template <int G, bool BF16>
__device__ __forceinline__ void zero_quad4(Quad4<G, BF16>& q) {
#pragma unroll
  for (int g = 0; g < G; ++g) q.raw[g] = u32x4{0u, 0u, 0u, 0u};
#pragma unroll
  for (int t = 0; t < Quad4<G, BF16>::TH; ++t) q.th[t] = 0.f;
}

// The Gram tiles of one vector slot: for each of its VE elements, the
// lane's group deltas (exact, fp64) go into every tile (I, J), I <= J.
template <int K, bool BF16>
__device__ __forceinline__ void gram_quad4(double (&acc)[Tiles4<K>::T], const u32x4 (&raw)[Tiles4<K>::G],
                                           const float (&th)[Vec<BF16>::VE], const bool (&act)[Tiles4<K>::G]) {
  constexpr int G = Tiles4<K>::G;
#pragma unroll
  for (int e = 0; e < Vec<BF16>::VE; ++e) {
    double d[G];
#pragma unroll
    for (int g = 0; g < G; ++g) d[g] = act[g] ? delta64<BF16>(raw[g], e, th[e]) : 0.0;
    int t = 0;
#pragma unroll
    for (int I = 0; I < G; ++I)
#pragma unroll
      for (int J = I; J < G; ++J, ++t) acc[t] = __builtin_amdgcn_mfma_f64_4x4x4f64(d[I], d[J], acc[t], 0, 0, 0);
  }
}

template <int K, bool BF16, bool NT>
__global__ __launch_bounds__(pass1_threads<K>()) void pass1_gram_mfma_kernel(const float* __restrict__ theta,
                                                                   ConstPtrs<K> reps, int64_t nvec,
                                                                   int64_t n,
                                                                   double* __restrict__ partials,
                                                                   PrevDecide prev,
                                                                   DecideParams prm) {
  static_assert(K > 8 && K <= 32, "MFMA Gram pass covers 8 < K <= 32");
  const int first = prev.partials ? 1 : 0;  // block 0 may take the previous unit's decision
  if (first && blockIdx.x == 0) {
    run_prev_decide<K, pass1_threads<K>()>(prev, prm);
    return;
  }
  const int b = static_cast<int>(blockIdx.x) - first;  // this block's partial row
  const int rows = static_cast<int>(gridDim.x) - first;
  constexpr int kDepth = kMfmaDepth<K>();
#include "gram_rows_mfma.inc"
}
// ---------------------------------------------------------------- decide

template <int K>
__global__ __launch_bounds__(kDecideThreads) void decide_kernel(const double* __restrict__ partials,
                                                                int rows, UnitRecord* __restrict__ rec,
                                                                DecideParams prm) {
  __shared__ double gram[K * (K + 1) / 2];
  __shared__ double scratch[kReduceLogical];
  const DecideState st = load_decide_state<K>(rec);
  reduce_partials<K, kDecideThreads>(partials, rows, gram, scratch);
  __syncthreads();
  if (threadIdx.x < 64) decide<K>(gram, rec, prm, st);
}

// The Gram of one unit as a plain vector (upper triangle, row by row): the
// decision kernel's own fixed-order reduction, written out instead of
// decided on, so that the shards of one module can add their Grams before a
// shared decision.
template <int K>
__global__ __launch_bounds__(kDecideThreads) void gram_reduce_kernel(const double* __restrict__ partials,
                                                                     int rows,
                                                                     double* __restrict__ gram_out) {
  __shared__ double gram[K * (K + 1) / 2];
  __shared__ double scratch[kReduceLogical];
  reduce_partials<K, kDecideThreads>(partials, rows, gram, scratch);
  __syncthreads();
  for (int p = threadIdx.x; p < K * (K + 1) / 2; p += kDecideThreads) gram_out[p] = gram[p];
}

// The decision from a Gram supplied by the caller (one wave).
template <int K>
__global__ __launch_bounds__(64) void decide_gram_kernel(const double* __restrict__ gram_in,
                                                         UnitRecord* __restrict__ rec,
                                                         DecideParams prm) {
  __shared__ double gram[K * (K + 1) / 2];
  const DecideState st = load_decide_state<K>(rec);
  for (int p = threadIdx.x; p < K * (K + 1) / 2; p += 64) gram[p] = gram_in[p];
  __syncthreads();
  decide<K>(gram, rec, prm, st);
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

// theta, b and the contributing replicas at vector v (nothing past the end).
template <int K, bool BF16, bool NT>
__device__ __forceinline__ void load_pass2(const float* theta, const float* mom,
                                           const u32x4* const (&src)[K], bool use, int64_t v,
                                           int64_t nvec, float (&th)[Vec<BF16>::VE],
                                           float (&b)[Vec<BF16>::VE], u32x4 (&raw)[K]) {
  if (v < nvec) {
    load_f32<Vec<BF16>::VE, NT>(theta, v, th);
    load_f32<Vec<BF16>::VE, NT>(mom, v, b);
    if (use) {
#pragma unroll
      for (int j = 0; j < K; ++j) raw[j] = ld16<NT>(src[j] + v);
    }
  }
}

// The update of one vector: weighted average, Nesterov, write-back.
template <int K, bool BF16, bool NT>
__device__ __forceinline__ void update_vector(float* theta, float* mom, const MutPtrs<K>& reps,
                                              const double (&c)[K], bool use, int64_t v,
                                              const float (&th)[Vec<BF16>::VE],
                                              const float (&b)[Vec<BF16>::VE],
                                              const u32x4 (&raw)[K], double lr, double rho) {
  constexpr int VE = Vec<BF16>::VE;
  double acc[VE];
#pragma unroll
  for (int e = 0; e < VE; ++e) acc[e] = 0.0;
  if (use) {
#pragma unroll
    for (int j = 0; j < K; ++j)
#pragma unroll
      for (int e = 0; e < VE; ++e) acc[e] = fma(c[j], delta64<BF16>(raw[j], e, th[e]), acc[e]);
  }
  float tn[VE], bn[VE];
#pragma unroll
  for (int e = 0; e < VE; ++e) nesterov(acc[e], th[e], b[e], lr, rho, tn[e], bn[e]);
  store_f32<VE, NT>(theta, v, tn);
  store_f32<VE, NT>(mom, v, bn);
  const u32x4 out = pack<BF16>(tn);
#pragma unroll
  for (int j = 0; j < K; ++j) st16<NT>(reinterpret_cast<u32x4*>(reps.p[j]) + v, out);
}

// One 16-byte vector of every buffer per thread, one one-wave block per 64
// vectors (a flat grid): the hardware dispatcher then keeps the in-flight
// window of each of the 2K+4 streams short and ordered (measured 5.5 TB/s
// here against 4.9 TB/s for a persistent grid-stride loop).  The launch
// reserves dynamic LDS so that six blocks at most run on a CU
// (update_pass_blocks_per_cu): fewer waves in flight serve this traffic
// faster.  Blocks are taken from the unit's end; forward order measured the
// same.
template <int K, bool BF16, bool NT>
__global__ __launch_bounds__(kPass2Threads) void pass2_update_kernel(float* __restrict__ theta,
                                                                float* __restrict__ mom,
                                                                MutPtrs<K> reps,
                                                                const UnitRecord* __restrict__ rec,
                                                                int64_t nvec, int64_t n, double lr,
                                                                double rho) {
  constexpr int VE = Vec<BF16>::VE;
  const int64_t v = static_cast<int64_t>(gridDim.x - 1 - blockIdx.x) * kPass2Threads + threadIdx.x;
  const int64_t tail = nvec * VE + threadIdx.x;
  const bool do_tail = blockIdx.x == 0 && tail < n;
  constexpr bool kRecFresh = false;  // written by the decision of an earlier launch

#include "update_vector_at.inc"
}

// The access pattern of pass 2 with no arithmetic: the same grid, block
// order and 16-byte accesses, reading theta, b and all K replicas and
// writing them all back (XOR with `flip`, zero at run time, keeps every
// store), so its time is what this traffic costs with nothing computed.
// Used to calibrate pass 2 against its own pattern, not by the method.
template <int K, bool BF16, bool NT>
__global__ __launch_bounds__(kPass2Threads) void update_pattern_probe_kernel(float* __restrict__ theta,
                                                                            float* __restrict__ mom,
                                                                            MutPtrs<K> reps, int64_t nvec,
                                                                            uint32_t flip) {
  const int64_t v = static_cast<int64_t>(gridDim.x - 1 - blockIdx.x) * kPass2Threads + threadIdx.x;
  if (v >= nvec) return;
  constexpr int H = Vec<BF16>::VE / 4;  // 16-byte vectors of theta (and of b) per replica vector
  u32x4 t[H], b[H], r[K];
  u32x4* tp = reinterpret_cast<u32x4*>(theta) + v * H;
  u32x4* bp = reinterpret_cast<u32x4*>(mom) + v * H;
#pragma unroll
  for (int h = 0; h < H; ++h) {
    t[h] = ld16<NT>(tp + h);
    b[h] = ld16<NT>(bp + h);
  }
#pragma unroll
  for (int j = 0; j < K; ++j) r[j] = ld16<NT>(reinterpret_cast<const u32x4*>(reps.p[j]) + v);
#pragma unroll
  for (int h = 0; h < H; ++h) {
    st16<NT>(tp + h, t[h] ^ flip);
    st16<NT>(bp + h, b[h] ^ flip);
  }
#pragma unroll
  for (int j = 0; j < K; ++j) st16<NT>(reinterpret_cast<u32x4*>(reps.p[j]) + v, r[j] ^ flip);
}

// ------------------------------------------- single-block units of a round

// A unit whose Gram pass is one block (at most 256 vectors) can be stepped
// whole by one block: its Gram row, the decision and the update pass, one
// after the other.  A round does that for up to kMaxSingleBlockUnits such
// units in one small launch, which may also carry the previous unit's
// decision (round_small_kernel).  The block runs the code of the unit's own
// three launches (pass 1 with one row, the decision, pass 2 with one vector
// per thread), included from the same fragments, so the results are the
// same bit for bit.  The partial row and the record are written and read
// back within the block: __syncthreads() orders global memory between the
// waves of one work-group (they share the CU's L1); the partials are read
// with non-temporal vector loads and the record with work-group-scope
// atomic loads (rec_load), never through the scalar cache.
template <int K>
struct SingleBlockUnit {
  float* theta;
  float* mom;
  void* reps[K];
  double* partials;
  UnitRecord* rec;
  int64_t n;
};

template <int K>
struct SingleBlockUnits {
  SingleBlockUnit<K> u[kMaxSingleBlockUnits];
  int count;
  double lr, rho;
};

template <int K, bool BF16, bool NT1, bool NT2, bool MFMA>
__device__ void single_block_unit(const SingleBlockUnit<K>& su, const DecideParams& prm, double lr,
                                  double rho) {
  constexpr int VE = Vec<BF16>::VE;
  const int64_t n = su.n;
  const int64_t nvec = n / VE;
  {  // pass 1: the unit's only Gram row
    constexpr bool NT = NT1;
    const float* __restrict__ theta = su.theta;
    ConstPtrs<K> reps;
#pragma unroll
    for (int j = 0; j < K; ++j) reps.p[j] = su.reps[j];
    double* __restrict__ partials = su.partials;
    const int b = 0, rows = 1;
    if constexpr (MFMA) {
      constexpr int kDepth = 2;  // a few trips at most: deeper prefetch only costs registers
#include "gram_rows_mfma.inc"
    } else {
      constexpr int NP = K * (K + 1) / 2;
#include "gram_rows_valu.inc"
    }
  }
  __syncthreads();
  run_prev_decide<K, pass1_threads<K>()>(PrevDecide{su.partials, 1, su.rec}, prm);
  __syncthreads();
  {  // pass 2: one vector per thread (nvec <= 256 <= the block's threads)
    constexpr bool NT = NT2;
    float* __restrict__ theta = su.theta;
    float* __restrict__ mom = su.mom;
    MutPtrs<K> reps;
#pragma unroll
    for (int j = 0; j < K; ++j) reps.p[j] = su.reps[j];
    const UnitRecord* rec = su.rec;
    const int64_t v = threadIdx.x;
    const int64_t tail = nvec * VE + threadIdx.x;
    const bool do_tail = tail < n;
    constexpr bool kRecFresh = true;  // written by this block's decision just above
#include "update_vector_at.inc"
  }
}

// Block 0 takes the decisions of up to two earlier units when prev0.partials
// is set; one block per single-block unit steps that unit.  The blocks have
// the pass-1 kernel's size, so a unit's Gram row is the one its own pass 1
// would write.
template <int K, bool BF16, bool NT1, bool NT2, bool MFMA>
__global__ __launch_bounds__(pass1_threads<K>()) void round_small_kernel(PrevDecide prev0, PrevDecide prev1,
                                                               DecideParams prm,
                                                               SingleBlockUnits<K> single) {
  const int first = prev0.partials ? 1 : 0;
  if (first && blockIdx.x == 0) {
    run_prev_decisions<K>(prev0, prev1, prm);
    return;
  }
  const int sb = static_cast<int>(blockIdx.x) - first;
  if (sb < single.count) single_block_unit<K, BF16, NT1, NT2, MFMA>(single.u[sb], prm, single.lr, single.rho);
}

// ------------------------------------------------------ one-pass mean step

// With every penalty component off (the plain DiLoCo outer step, the paper's
// "w/o ALL" ablation), the weights are 1/K whatever the norms are, so the
// average, Nesterov and the write-back need no earlier pass: one kernel reads
// theta, b and the K replicas once and writes theta', b' and the replicas.
// The norms G_j and ||Delta_bar|| are still summed on the way (per-block
// partials, reduced by fused_finish_kernel) for the step's record, and the
// unit is marked for that reduction.  A block owns V*kFusedThreads
// consecutive vectors; a thread loads its V vectors of every buffer before
// computing, so V*(K+2) 16-byte loads are in flight per thread (V = 2 for
// bf16 replicas measured best here: one vector leaves the block's closing
// reduction exposed, four cost occupancy).
template <int K, bool BF16, bool NT, int V>
__global__ __launch_bounds__(kFusedThreads) void fused_mean_kernel(float* __restrict__ theta,
                                                                   float* __restrict__ mom,
                                                                   MutPtrs<K> reps,
                                                                   double* __restrict__ partials,
                                                                   UnitRecord* __restrict__ rec,
                                                                   int64_t nvec, int64_t n,
                                                                   double lr, double rho) {
  constexpr int VE = Vec<BF16>::VE;
  constexpr double inv_k = 1.0 / K;
  const int b = blockIdx.x;
  double sq[K + 1];  // sum of Delta_j^2 per worker, then of Delta_bar^2
#pragma unroll
  for (int p = 0; p <= K; ++p) sq[p] = 0.0;

  {
    const int64_t base = static_cast<int64_t>(b) * V * kFusedThreads + threadIdx.x;
    float th[V][VE], bm[V][VE];
    u32x4 raw[V][K];
#pragma unroll
    for (int u = 0; u < V; ++u) {
      const int64_t v = base + u * kFusedThreads;
      if (v < nvec) {
        load_f32<VE, NT>(theta, v, th[u]);
        load_f32<VE, NT>(mom, v, bm[u]);
#pragma unroll
        for (int j = 0; j < K; ++j) raw[u][j] = ld16<NT>(reinterpret_cast<const u32x4*>(reps.p[j]) + v);
      }
    }
#pragma unroll
    for (int u = 0; u < V; ++u) {
      const int64_t v = base + u * kFusedThreads;
      if (v < nvec) {
        float tn[VE], bn[VE];
#pragma unroll
        for (int e = 0; e < VE; ++e) {
          double sum = 0.0;
#pragma unroll
          for (int j = 0; j < K; ++j) {
            const double d = delta64<BF16>(raw[u][j], e, th[u][e]);
            sq[j] = fma(d, d, sq[j]);
            sum += d;
          }
          const double dbar = sum * inv_k;  // Eq. 3 with w_j = 1/K
          sq[K] = fma(dbar, dbar, sq[K]);
          nesterov(dbar, th[u][e], bm[u][e], lr, rho, tn[e], bn[e]);
        }
        store_f32<VE, NT>(theta, v, tn);
        store_f32<VE, NT>(mom, v, bn);
        const u32x4 out = pack<BF16>(tn);
#pragma unroll
        for (int j = 0; j < K; ++j) st16<NT>(reinterpret_cast<u32x4*>(reps.p[j]) + v, out);
      }
    }
  }
  const int64_t tail = nvec * VE + threadIdx.x;  // the last n - nvec*VE elements
  if (b == 0 && tail < n) {
    const float t0 = theta[tail];
    double sum = 0.0;
#pragma unroll
    for (int j = 0; j < K; ++j) {
      const double d = static_cast<double>(load_scalar<BF16>(reps.p[j], tail)) - static_cast<double>(t0);
      sq[j] = fma(d, d, sq[j]);
      sum += d;
    }
    const double dbar = sum * inv_k;
    sq[K] = fma(dbar, dbar, sq[K]);
    float tn, bn;
    nesterov(dbar, t0, mom[tail], lr, rho, tn, bn);
    theta[tail] = tn;
    mom[tail] = bn;
#pragma unroll
    for (int j = 0; j < K; ++j) store_scalar<BF16>(reps.p[j], tail, tn);
  }

  // block sums in a fixed order: wave butterfly, then the waves in order
  constexpr int kWaves = kFusedThreads / 64;
  __shared__ double red[kWaves][K + 1];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int p = 0; p <= K; ++p) {
    const double t = wave_sum(sq[p]);
    if (lane == 0) red[wave][p] = t;
  }
  __syncthreads();
  if (threadIdx.x <= K) {  // the block's K + 1 sums, contiguous
    double t = red[0][threadIdx.x];
#pragma unroll
    for (int w = 1; w < kWaves; ++w) t += red[w][threadIdx.x];
    partials[static_cast<int64_t>(b) * (K + 1) + threadIdx.x] = t;
  }
  if (b == 0 && threadIdx.x == 0) rec->finish_pending = 1;
}

// The records of one-pass steps: G_j and ||Delta_bar|| from each unit's
// partials (in a fixed order), w_j = 1/K, beta = 1.  One block per unit of
// `table`; units whose fused pass has not run since their last record are
// skipped, so a round can take all its units' reductions in one launch after
// its last fused pass.  Nothing is masked in this mode: a non-finite replica
// shows up as a non-finite G_j (and in theta).
template <int K>
__global__ __launch_bounds__(kDecideThreads) void fused_finish_kernel(const FinishEntry* __restrict__ table) {
  const FinishEntry ent = table[blockIdx.x];
  UnitRecord* rec = ent.rec;
  if (!rec->finish_pending) return;  // block-uniform
  const double* partials = ent.partials;
  const int rows = ent.rows;
  constexpr int NV = K + 1;
  // The partials are rows x NV contiguous doubles.  Thread t reads the flat
  // array at t, t + S, t + 2S, ... with S a multiple of NV, so it always
  // reads column t % NV and a wave's loads are contiguous; U loads per
  // thread are in flight at a time.  The S threads' sums are then added per
  // column in thread order (a fixed order).
  constexpr int S = NV * (kDecideThreads / NV);
  constexpr int U = 16;
  __shared__ double part[kDecideThreads];
  __shared__ double tot[NV];
  const int64_t total = static_cast<int64_t>(rows) * NV;
  double s = 0.0;
  if (threadIdx.x < S) {
    for (int64_t i = threadIdx.x; i < total; i += int64_t(S) * U) {
      double v[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int64_t idx = i + int64_t(u) * S;
        v[u] = idx < total ? partials[idx] : 0.0;
      }
#pragma unroll
      for (int u = 0; u < U; ++u) s += v[u];
    }
  }
  part[threadIdx.x] = s;
  __syncthreads();
  if (threadIdx.x < NV) {
    double t = 0.0;
    for (int k = threadIdx.x; k < S; k += NV) t += part[k];
    tot[threadIdx.x] = t;
  }
  __syncthreads();
  if (threadIdx.x < K) {
    rec->norm[threadIdx.x] = sqrt(tot[threadIdx.x]);
    rec->weight[threadIdx.x] = 1.0 / K;
    rec->coef[threadIdx.x] = 1.0 / K;
    rec->src[threadIdx.x] = threadIdx.x;
    rec->anomalous[threadIdx.x] = 0;
  }
  if (threadIdx.x == 0) {
    rec->synced_norm = sqrt(tot[K]);
    rec->clip_coef = 1.0;
    rec->use_deltas = 1;
    rec->rollback = 0;
    rec->z_tested = 0;
    rec->stepped = 1;
    rec->round = rec->round + 1;
    rec->finish_pending = 0;
  }
}

// ------------------------------------------------------------ copy probe

template <int U, bool NT>
__global__ __launch_bounds__(kThreads) void copy_kernel(u32x4* __restrict__ dst,
                                                       const u32x4* __restrict__ src,
                                                       int64_t nvec) {
  const int64_t stride = static_cast<int64_t>(gridDim.x) * kThreads;
  for (int64_t v = static_cast<int64_t>(blockIdx.x) * kThreads + threadIdx.x; v < nvec; v += stride * U) {
    u32x4 x[U];
#pragma unroll
    for (int u = 0; u < U; ++u)
      if (u == 0 || v + u * stride < nvec) x[u] = ld16<NT>(src + v + u * stride);
#pragma unroll
    for (int u = 0; u < U; ++u)
      if (u == 0 || v + u * stride < nvec) st16<NT>(dst + v + u * stride, x[u]);
  }
}

}  // namespace

// ------------------------------------------------------------ launchers

// Cache policy of the streaming kernels: both passes touch every byte once;
// non-temporal accesses measured ~15% faster for pass 1 and ~5% for pass 2.
constexpr bool kNT1 = true;
constexpr bool kNTMfma = false;  // see pass1_gram_mfma_kernel
constexpr bool kNT2 = true;

namespace {

// Pass 1 for this K: VALU accumulators up to K = 8, matrix cores above.
template <int K, bool BF16>
constexpr auto pass1_kernel() {
  if constexpr (K <= 8)
    return pass1_gram_kernel<K, BF16, kNT1>;
  else
    return pass1_gram_mfma_kernel<K, BF16, kNTMfma>;
}

template <int K, bool BF16>
hipError_t pass1_launch(int rows, const float* theta, const void* const* reps, int64_t n,
                        double* partials, const double* prev_partials, int prev_rows,
                        UnitRecord* prev_rec, const DecideParams& prm, hipStream_t stream) {
  ConstPtrs<K> rp;
  for (int j = 0; j < K; ++j) rp.p[j] = reps[j];
  const int64_t nvec = n / Vec<BF16>::VE;
  const PrevDecide prev{prev_partials, prev_rows, prev_rec};
  const int blocks = rows + (prev_partials ? 1 : 0);
  hipLaunchKernelGGL((pass1_kernel<K, BF16>()), dim3(blocks), dim3(pass1_threads<K>()), 0, stream, theta, rp,
                     nvec, n, partials, prev, prm);
  return hipGetLastError();
}

// Block 0's decisions: prev[0..nprev), nprev <= 2.
inline void prev_decisions(const DecideDesc* prev, int nprev, PrevDecide& p0, PrevDecide& p1) {
  p0 = nprev > 0 ? PrevDecide{prev[0].partials, prev[0].rows, prev[0].rec} : PrevDecide{nullptr, 0, nullptr};
  p1 = nprev > 1 ? PrevDecide{prev[1].partials, prev[1].rows, prev[1].rec} : PrevDecide{nullptr, 0, nullptr};
}

template <int K, bool BF16>
Pass1Part<K> pass1_part(const Pass1Desc* unit, int count, int i) {
  Pass1Part<K> part{};
  if (i >= count) return part;  // rows 0: no unit
  const Pass1Desc& d = unit[i];
  part.theta = d.theta;
  for (int j = 0; j < K; ++j) part.reps.p[j] = d.n > 0 ? d.reps[j] : nullptr;
  part.nvec = d.n / Vec<BF16>::VE;
  part.n = d.n;
  part.partials = d.partials;
  part.rows = d.rows;
  return part;
}

template <int K, bool BF16>
hipError_t pass1_pair_launch(const Pass1Desc* unit, int count, const DecideDesc* prev, int nprev,
                             const DecideParams& prm, hipStream_t stream) {
  if constexpr (K > 8) {
    return hipErrorInvalidValue;  // the matrix-core Gram pass runs one unit per launch
  } else {
    PrevDecide p0, p1;
    prev_decisions(prev, nprev, p0, p1);
    const Pass1Part<K> u0 = pass1_part<K, BF16>(unit, count, 0);
    const Pass1Part<K> u1 = pass1_part<K, BF16>(unit, count, 1);
    const int blocks = (nprev > 0 ? 1 : 0) + std::max(u0.rows, u1.rows);
    if (count == 2)
      hipLaunchKernelGGL((pass1_gram_pair_kernel<K, BF16, kNT1, 2>), dim3(blocks), dim3(pass1_threads<K>()),
                         0, stream, u0, u1, p0, p1, prm);
    else
      hipLaunchKernelGGL((pass1_gram_pair_kernel<K, BF16, kNT1, 1>), dim3(blocks), dim3(pass1_threads<K>()),
                         0, stream, u0, u1, p0, p1, prm);
    return hipGetLastError();
  }
}

template <int K, bool BF16>
hipError_t round_small_launch(const DecideDesc* prev, int nprev, const DecideParams& prm,
                              const SingleBlockDesc* unit, int count, double lr, double rho,
                              hipStream_t stream) {
  PrevDecide p0, p1;
  prev_decisions(prev, nprev, p0, p1);
  SingleBlockUnits<K> single{};
  single.count = count;
  single.lr = lr;
  single.rho = rho;
  for (int i = 0; i < count; ++i) {
    const SingleBlockDesc& d = unit[i];
    single.u[i].theta = d.theta;
    single.u[i].mom = d.mom;
    for (int j = 0; j < K; ++j) single.u[i].reps[j] = d.n > 0 ? d.reps[j] : nullptr;
    single.u[i].partials = d.partials;
    single.u[i].rec = d.rec;
    single.u[i].n = d.n;
  }
  const int blocks = (nprev > 0 ? 1 : 0) + count;
  if (blocks == 0) return hipSuccess;
  constexpr bool kMfma = K > 8;
  hipLaunchKernelGGL((round_small_kernel<K, BF16, kMfma ? kNTMfma : kNT1, kNT2, kMfma>), dim3(blocks),
                     dim3(pass1_threads<K>()), 0, stream, p0, p1, prm, single);
  return hipGetLastError();
}

template <int K>
hipError_t decide_launch(const double* partials, int rows, UnitRecord* rec, const DecideParams& prm,
                         hipStream_t stream) {
  hipLaunchKernelGGL((decide_kernel<K>), dim3(1), dim3(kDecideThreads), 0, stream, partials, rows, rec,
                     prm);
  return hipGetLastError();
}

template <int K>
hipError_t gram_reduce_launch(const double* partials, int rows, double* gram, hipStream_t stream) {
  hipLaunchKernelGGL((gram_reduce_kernel<K>), dim3(1), dim3(kDecideThreads), 0, stream, partials, rows,
                     gram);
  return hipGetLastError();
}

template <int K>
hipError_t decide_gram_launch(const double* gram, UnitRecord* rec, const DecideParams& prm,
                              hipStream_t stream) {
  hipLaunchKernelGGL((decide_gram_kernel<K>), dim3(1), dim3(64), 0, stream, gram, rec, prm);
  return hipGetLastError();
}

template <int K, bool BF16>
hipError_t pattern_probe_launch(int blocks, int lds, float* theta, float* mom, void* const* reps, int64_t n,
                                hipStream_t stream) {
  MutPtrs<K> rp;
  for (int j = 0; j < K; ++j) rp.p[j] = reps[j];
  const int64_t nvec = n / Vec<BF16>::VE;
  hipLaunchKernelGGL((update_pattern_probe_kernel<K, BF16, kNT2>), dim3(blocks), dim3(kPass2Threads), lds, stream,
                     theta, mom, rp, nvec, 0u);
  return hipGetLastError();
}

template <int K, bool BF16>
hipError_t pass2_launch(int blocks, int lds, float* theta, float* mom, void* const* reps,
                        const UnitRecord* rec, int64_t n, double lr, double rho, hipStream_t stream) {
  MutPtrs<K> rp;
  for (int j = 0; j < K; ++j) rp.p[j] = reps[j];
  const int64_t nvec = n / Vec<BF16>::VE;
  hipLaunchKernelGGL((pass2_update_kernel<K, BF16, kNT2>), dim3(blocks), dim3(kPass2Threads), lds, stream, theta,
                     mom, rp, rec, nvec, n, lr, rho);
  return hipGetLastError();
}

// Vectors per thread of the one-pass kernel (measured: two 16-byte vectors
// of bf16 replicas, one of fp32; one above K = 16, where two would hold
// 2K 16-byte registers of replica data per lane).
template <int K, bool BF16>
constexpr int fused_v() {
  return BF16 && K <= 16 ? 2 : 1;
}

template <int K, bool BF16>
hipError_t fused_mean_launch(int rows, int lds, float* theta, float* mom, void* const* reps, double* partials,
                             UnitRecord* rec, int64_t n, double lr, double rho, hipStream_t stream) {
  MutPtrs<K> rp;
  for (int j = 0; j < K; ++j) rp.p[j] = reps[j];
  const int64_t nvec = n / Vec<BF16>::VE;
  hipLaunchKernelGGL((fused_mean_kernel<K, BF16, kNT2, fused_v<K, BF16>()>), dim3(rows), dim3(kFusedThreads),
                     lds, stream, theta, mom, rp, partials, rec, nvec, n, lr, rho);
  return hipGetLastError();
}

template <int K>
hipError_t fused_finish_launch(const FinishEntry* table, int units, hipStream_t stream) {
  hipLaunchKernelGGL((fused_finish_kernel<K>), dim3(units), dim3(kDecideThreads), 0, stream, table);
  return hipGetLastError();
}

template <typename Kern>
int occupancy(Kern kernel, int threads) {
  int blocks = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&blocks, kernel, threads, 0) != hipSuccess ||
      blocks < 1)
    blocks = 1;
  return blocks;
}

template <int K>
struct Launchers {
  static hipError_t pass1(bool bf16, int rows, const float* theta, const void* const* reps, int64_t n,
                          double* partials, const double* prev_partials, int prev_rows, UnitRecord* prev_rec,
                          const DecideParams& prm, hipStream_t stream) {
    return bf16 ? pass1_launch<K, true>(rows, theta, reps, n, partials, prev_partials, prev_rows, prev_rec, prm,
                                        stream)
                : pass1_launch<K, false>(rows, theta, reps, n, partials, prev_partials, prev_rows, prev_rec, prm,
                                         stream);
  }
  static hipError_t pass1_pair(bool bf16, const Pass1Desc* unit, int count, const DecideDesc* prev, int nprev,
                               const DecideParams& prm, hipStream_t stream) {
    return bf16 ? pass1_pair_launch<K, true>(unit, count, prev, nprev, prm, stream)
                : pass1_pair_launch<K, false>(unit, count, prev, nprev, prm, stream);
  }
  static hipError_t round_small(bool bf16, const DecideDesc* prev, int nprev, const DecideParams& prm,
                                const SingleBlockDesc* unit, int count, double lr, double rho,
                                hipStream_t stream) {
    return bf16 ? round_small_launch<K, true>(prev, nprev, prm, unit, count, lr, rho, stream)
                : round_small_launch<K, false>(prev, nprev, prm, unit, count, lr, rho, stream);
  }
  static hipError_t pass2(bool bf16, int blocks, int lds, float* theta, float* mom, void* const* reps,
                          const UnitRecord* rec, int64_t n, double lr, double rho, hipStream_t stream) {
    return bf16 ? pass2_launch<K, true>(blocks, lds, theta, mom, reps, rec, n, lr, rho, stream)
                : pass2_launch<K, false>(blocks, lds, theta, mom, reps, rec, n, lr, rho, stream);
  }
  static hipError_t pattern_probe(bool bf16, int blocks, int lds, float* theta, float* mom, void* const* reps,
                                  int64_t n, hipStream_t stream) {
    return bf16 ? pattern_probe_launch<K, true>(blocks, lds, theta, mom, reps, n, stream)
                : pattern_probe_launch<K, false>(blocks, lds, theta, mom, reps, n, stream);
  }
  static hipError_t fused_mean(bool bf16, int rows, int lds, float* theta, float* mom, void* const* reps,
                               double* partials, UnitRecord* rec, int64_t n, double lr, double rho,
                               hipStream_t stream) {
    return bf16 ? fused_mean_launch<K, true>(rows, lds, theta, mom, reps, partials, rec, n, lr, rho, stream)
                : fused_mean_launch<K, false>(rows, lds, theta, mom, reps, partials, rec, n, lr, rho, stream);
  }
  static int pass1_blocks_per_cu(bool bf16) {
    return bf16 ? occupancy(pass1_kernel<K, true>(), pass1_threads<K>())
                : occupancy(pass1_kernel<K, false>(), pass1_threads<K>());
  }
};

// The set of K, or nullptr when K lies outside this object's range (the
// discarded branch instantiates nothing).
template <int K>
const KernelSet* set_if_in_range() {
  if constexpr (K >= EDIT_K_FIRST && K <= EDIT_K_LAST) {
    static constexpr KernelSet set{
        &Launchers<K>::pass1,          &Launchers<K>::pass1_pair,     &Launchers<K>::round_small,
        &decide_launch<K>,             &gram_reduce_launch<K>,        &decide_gram_launch<K>,
        &Launchers<K>::pass2,          &Launchers<K>::fused_mean,     &fused_finish_launch<K>,
        &Launchers<K>::pass1_blocks_per_cu, &Launchers<K>::pattern_probe, fused_v<K, true>(),
        fused_v<K, false>()};
    return &set;
  } else {
    return nullptr;
  }
}

}  // namespace

#define EDIT_FOR_EACH_K(X)                                                                       \
  X(1) X(2) X(3) X(4) X(5) X(6) X(7) X(8) X(9) X(10) X(11) X(12) X(13) X(14) X(15) X(16) X(17)   \
  X(18) X(19) X(20) X(21) X(22) X(23) X(24) X(25) X(26) X(27) X(28) X(29) X(30) X(31) X(32)

const KernelSet* EDIT_KERNEL_SET_FN(EDIT_K_FIRST)(int K) {
  switch (K) {
#define EDIT_CASE(KK) \
  case KK:            \
    return set_if_in_range<KK>();
    EDIT_FOR_EACH_K(EDIT_CASE)
#undef EDIT_CASE
    default:
      return nullptr;
  }
}

#if EDIT_K_FIRST == 1  // the copy probe is compiled into one object only
constexpr int kUnrollCopy = 1;
constexpr bool kNTCopy = false;

hipError_t launch_copy(void* dst, const void* src, int64_t nbytes, int blocks, hipStream_t stream) {
  hipLaunchKernelGGL((copy_kernel<kUnrollCopy, kNTCopy>), dim3(blocks), dim3(kThreads), 0, stream,
                     reinterpret_cast<u32x4*>(dst), reinterpret_cast<const u32x4*>(src), nbytes / 16);
  return hipGetLastError();
}
#endif

}  // namespace edit
