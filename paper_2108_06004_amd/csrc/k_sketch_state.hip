// k_sketch_state.hip -- momentum and error accumulation kept in the merged sketch.
//
// The Count Sketch is linear (Sec. III-A: S(a + b) = S(a) + S(b)), so momentum and error
// accumulation can be carried inside it instead of in d-vectors per worker (Sec. II,
// sketching paragraph). One step, after the workers' sketches of g are merged into S:
//   U <- fl(fl(rho U) + S),  E <- fl(E + U)                    per cell, fp32, no FMA
//   Top_k = the k largest |estimate of E|, ties to the lower index (the usual selection)
//   Delta_i = estimate of E at i, for i in Top_k               (the step's values)
//   E <- fl(E - D) on every cell D touches, D = S(Delta) summed per cell in fp64 and
//        rounded once; U <- 0 on those cells when momentum is reset
// The subtraction runs in three passes over the k*r (coordinate, row) pairs: clear the
// touched cells' fp64 accumulators and claim bits, add the signed values (fp64 atomics),
// and let the first pair to claim each cell apply it.
#include "gs_internal.hpp"

namespace gs {
namespace {

constexpr int kBlock = 256;

int grid_for(int64_t work_items, int per_block, int cap) {
  int64_t b = (work_items + per_block - 1) / per_block;
  if (b < 1) b = 1;
  if (b > cap) b = cap;
  return (int)b;
}

__global__ void __launch_bounds__(kBlock) k_sketch_mom(const float* __restrict__ S, float* __restrict__ U,
                                                       float* __restrict__ E, int64_t rc, float rho) {
  const int64_t stride = (int64_t)gridDim.x * kBlock;
  for (int64_t e = (int64_t)blockIdx.x * kBlock + threadIdx.x; e < rc; e += stride) {
    const float m = rho * U[e];
    const float u = m + S[e];
    U[e] = u;
    E[e] = E[e] + u;
  }
}

template <int R>
__global__ void __launch_bounds__(kBlock) k_values_at(HashSet hs, const float* __restrict__ E,
                                                      const int32_t* __restrict__ idx, int64_t k,
                                                      float* __restrict__ values) {
  RowConst kr[R];
#pragma unroll
  for (int j = 0; j < R; ++j) kr[j] = row_const(hs, j);
  const int64_t stride = (int64_t)gridDim.x * kBlock;
  for (int64_t t = (int64_t)blockIdx.x * kBlock + threadIdx.x; t < k; t += stride)
    values[t] = estimate_val<R>(kr, E, (uint32_t)idx[t]);
}

// Pair p = t * r + j: row j of selected coordinate idx[t].
__device__ __forceinline__ int64_t pair_cell(const HashSet& hs, const int32_t* __restrict__ idx, int64_t p,
                                             uint32_t& sflip) {
  const int64_t t = p / hs.r;
  const int j = (int)(p - t * hs.r);
  uint32_t col;
  hash_ij(hs, j, (uint32_t)idx[t], col, sflip);
  return (int64_t)j * hs.c + col;
}

__global__ void __launch_bounds__(kBlock) k_sub_clear(HashSet hs, const int32_t* __restrict__ idx, int64_t n_pairs,
                                                      double* __restrict__ acc, uint32_t* __restrict__ claim) {
  const int64_t stride = (int64_t)gridDim.x * kBlock;
  for (int64_t p = (int64_t)blockIdx.x * kBlock + threadIdx.x; p < n_pairs; p += stride) {
    uint32_t sflip;
    const int64_t cell = pair_cell(hs, idx, p, sflip);
    acc[cell] = 0.0;
    atomicAnd(&claim[cell >> 5], ~(1u << (cell & 31)));
  }
}

__global__ void __launch_bounds__(kBlock) k_sub_add(HashSet hs, const int32_t* __restrict__ idx, int64_t n_pairs,
                                                    const float* __restrict__ values, double* __restrict__ acc) {
  const int64_t stride = (int64_t)gridDim.x * kBlock;
  for (int64_t p = (int64_t)blockIdx.x * kBlock + threadIdx.x; p < n_pairs; p += stride) {
    uint32_t sflip;
    const int64_t cell = pair_cell(hs, idx, p, sflip);
    atomicAdd(&acc[cell], (double)apply_sign(values[p / hs.r], sflip));
  }
}

__global__ void __launch_bounds__(kBlock) k_sub_apply(HashSet hs, const int32_t* __restrict__ idx, int64_t n_pairs,
                                                      const double* __restrict__ acc, uint32_t* __restrict__ claim,
                                                      float* __restrict__ U, float* __restrict__ E,
                                                      int reset_momentum) {
  const int64_t stride = (int64_t)gridDim.x * kBlock;
  for (int64_t p = (int64_t)blockIdx.x * kBlock + threadIdx.x; p < n_pairs; p += stride) {
    uint32_t sflip;
    const int64_t cell = pair_cell(hs, idx, p, sflip);
    const uint32_t bit = 1u << (cell & 31);
    if ((atomicOr(&claim[cell >> 5], bit) & bit) == 0u) {
      E[cell] = E[cell] - (float)acc[cell];
      if (reset_momentum) U[cell] = 0.0f;
    }
  }
}

}  // namespace

hipError_t launch_sketch_state(gs_ctx* x, hipStream_t s, const float* merged, float* U, float* E, int64_t k,
                               int32_t* idx, float* values) {
  const int64_t rc = (int64_t)x->r * x->c;
  hipLaunchKernelGGL(k_sketch_mom, dim3(grid_for(rc, kBlock, 8 * x->num_cus)), dim3(kBlock), 0, s, merged, U, E, rc,
                     x->rho);
  hipError_t e = launch_unsketch_topk(x, s, E, k, nullptr, idx);
  stage_mark(x, s, 4);
  if (e != hipSuccess) return e;
  const dim3 gk(grid_for(k, kBlock, 4 * x->num_cus)), block(kBlock);
  switch (x->r) {
#define GS_R_CASE(RR) \
  case RR: hipLaunchKernelGGL(k_values_at<RR>, gk, block, 0, s, x->hs, E, idx, k, values); break;
    GS_R_CASE(1) GS_R_CASE(2) GS_R_CASE(3) GS_R_CASE(4) GS_R_CASE(5) GS_R_CASE(6) GS_R_CASE(7) GS_R_CASE(8)
    GS_R_CASE(9) GS_R_CASE(10) GS_R_CASE(11) GS_R_CASE(12) GS_R_CASE(13) GS_R_CASE(14) GS_R_CASE(15) GS_R_CASE(16)
#undef GS_R_CASE
    default: return hipErrorInvalidValue;
  }
  // fp64 cell accumulators and claim bits: context scratch free at this point of the step
  double* acc = x->use_pull ? x->partial : x->acc64;
  uint32_t* claim = x->heavy;
  const int64_t n_pairs = k * x->r;
  const dim3 gp(grid_for(n_pairs, kBlock, 8 * x->num_cus));
  hipLaunchKernelGGL(k_sub_clear, gp, block, 0, s, x->hs, idx, n_pairs, acc, claim);
  hipLaunchKernelGGL(k_sub_add, gp, block, 0, s, x->hs, idx, n_pairs, values, acc);
  hipLaunchKernelGGL(k_sub_apply, gp, block, 0, s, x->hs, idx, n_pairs, acc, claim, U, E, x->reset_momentum);
  stage_mark(x, s, 5);
  return hipGetLastError();
}

}  // namespace gs
