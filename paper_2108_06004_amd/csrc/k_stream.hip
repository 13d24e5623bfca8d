// k_stream.hip -- streaming kernels of the hot path: accumulation, table clearing, Count
// Sketch insertion, binomial-tree merge, exact-value gather with reset.
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

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

// ------------------------------------------------------------------------------------
// Momentum + error accumulation (Sec. II sketching paragraph): u = rho*u + g; v = v + u,
// each operation rounded to fp32 (the library is built with -ffp-contract=off, so no
// multiply-add is fused). The update is elementwise, so the [P][d] arrays are streamed as
// one flat vector of n = P*d floats, four per lane.

typedef float f4 __attribute__((ext_vector_type(4)));

// Each wave takes U = 4 consecutive chunks of 64 quads (4 KB of each array) per pass, all
// its loads in flight together, and every load and store is non-temporal (the streams are
// read and written once): as the interleaved accumulation, which these settings brought to
// the part's stream rate; the quads past the last whole group go one per lane.
__global__ void __launch_bounds__(kBlock) k_accumulate4(const f4* __restrict__ g, f4* __restrict__ u,
                                                        f4* __restrict__ v, int64_t n4, float rho) {
  constexpr int U = 4;
  const int lane = threadIdx.x & 63;
  const int64_t ngr = n4 / (64 * U);
  const int64_t wstride = (int64_t)gridDim.x * (kBlock / 64);
  const int64_t w0 = (int64_t)blockIdx.x * (kBlock / 64) + (threadIdx.x >> 6);
  for (int64_t gr = w0; gr < ngr; gr += wstride) {
    f4 gg[U], uu[U], vv[U];
#pragma unroll
    for (int m = 0; m < U; ++m) {
      const int64_t t = (gr * U + m) * 64 + lane;
      gg[m] = __builtin_nontemporal_load(g + t);
      uu[m] = __builtin_nontemporal_load(u + t);
      vv[m] = __builtin_nontemporal_load(v + t);
    }
#pragma unroll
    for (int m = 0; m < U; ++m) {
      const int64_t t = (gr * U + m) * 64 + lane;
      uu[m] = rho * uu[m] + gg[m];
      vv[m] = vv[m] + uu[m];
      __builtin_nontemporal_store(uu[m], u + t);
      __builtin_nontemporal_store(vv[m], v + t);
    }
  }
  const int64_t stride = (int64_t)gridDim.x * kBlock;
  for (int64_t t = ngr * U * 64 + (int64_t)blockIdx.x * kBlock + threadIdx.x; t < n4; t += stride) {
    const f4 gg = g[t];
    f4 uu = u[t], vv = v[t];
    uu = rho * uu + gg;
    vv = vv + uu;
    u[t] = uu;
    v[t] = vv;
  }
}

__global__ void __launch_bounds__(kBlock) k_accumulate1(const float* __restrict__ g, float* __restrict__ u,
                                                        float* __restrict__ v, int64_t lo, int64_t n, float rho) {
  const int64_t stride = (int64_t)gridDim.x * kBlock;
  for (int64_t t = lo + (int64_t)blockIdx.x * kBlock + threadIdx.x; t < n; t += stride) {
    const float un = rho * u[t] + g[t];
    u[t] = un;
    v[t] = v[t] + un;
  }
}

// Worker-interleaved state (u, v rows of PP = 4G floats per coordinate; g stays [P][d]).
// A wave covers CW = 64/G consecutive coordinates: lane l takes coordinate base + l/G and
// the 16-byte group h = l%G of its row (workers 4h..4h+3), so consecutive lanes read and
// write consecutive 16-byte pieces of u and v; the four gradient values come from four
// worker rows of g (4-byte loads, 4*CW bytes contiguous per row and wave). Each pass a wave
// takes U consecutive chunks (four, eight for G = 4), all in flight together, so when CW*4
// bytes is less than a 128-byte line (G = 3, 4) the rest of the line is read by the wave's
// next instruction.
// The chunks past the last group run one at a time, and with RAGGED (d not a multiple
// of CW) the first wave then takes the partial last chunk, whose lanes past d take no
// coordinate. The non-ragged form is kept free of that code: the compiler schedules this loop
// differently when it is there, and the schedule it picks for G = 2 without it measured 2%
// faster (0.650 against 0.662 ms at d = 25.6M x 8). For G = 4 a group is eight chunks, and its
// loads are all issued before any arithmetic (a scheduling barrier): at d = 66M x 16 the
// barrier took 3.97 to 3.89 ms and the eight chunks a further 1-2% (3.38 to 3.34 ms on a
// faster part); eight chunks for G = 1, 2, or the barrier there, measured slower.
template <int G, bool RAGGED>
__global__ void __launch_bounds__(kBlock) k_accumulate_il(const float* __restrict__ g, float* __restrict__ u,
                                                          float* __restrict__ v, int64_t d, float rho) {
  constexpr int CW = 64 / G;
  constexpr int PP = 4 * G;
  constexpr int U = G == 4 ? 8 : 4;
  const int lane = threadIdx.x & 63;
  if (lane >= CW * G) return;  // G = 3: one idle lane per wave (no barrier below)
  const int h = lane % G;
  const int64_t sub = lane / G;
  const int64_t nch = d / CW;  // full chunks
  const int64_t wstride = (int64_t)gridDim.x * (kBlock / 64);
  const int64_t ngr = nch / U;  // groups of U consecutive chunks, one group per wave and pass
  const int64_t w0 = (int64_t)blockIdx.x * (kBlock / 64) + (threadIdx.x >> 6);
  for (int64_t gr = w0; gr < ngr; gr += wstride) {
    f4 gg[U], uu[U], ww[U];
#pragma unroll
    for (int m = 0; m < U; ++m) {
      const int64_t i = (gr * U + m) * CW + sub;
      const float* gq = g + (int64_t)(4 * h) * d + i;
      gg[m].x = __builtin_nontemporal_load(gq);
      gg[m].y = __builtin_nontemporal_load(gq + d);
      gg[m].z = __builtin_nontemporal_load(gq + 2 * d);
      gg[m].w = __builtin_nontemporal_load(gq + 3 * d);
      uu[m] = __builtin_nontemporal_load(reinterpret_cast<const f4*>(u + i * PP) + h);
      ww[m] = __builtin_nontemporal_load(reinterpret_cast<const f4*>(v + i * PP) + h);
    }
    if constexpr (G == 4) __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int m = 0; m < U; ++m) {
      const int64_t i = (gr * U + m) * CW + sub;
      uu[m] = rho * uu[m] + gg[m];
      ww[m] = ww[m] + uu[m];
      __builtin_nontemporal_store(uu[m], reinterpret_cast<f4*>(u + i * PP) + h);
      __builtin_nontemporal_store(ww[m], reinterpret_cast<f4*>(v + i * PP) + h);
    }
  }
  for (int64_t ch = ngr * U + w0; ch < nch; ch += wstride) {  // chunks past the last group
    const int64_t i = ch * CW + sub;
    const float* gq = g + (int64_t)(4 * h) * d + i;
    f4 gg;
    gg.x = gq[0];
    gg.y = gq[d];
    gg.z = gq[2 * d];
    gg.w = gq[3 * d];
    f4* up = reinterpret_cast<f4*>(u + i * PP) + h;
    f4* vp = reinterpret_cast<f4*>(v + i * PP) + h;
    f4 uu = *up, ww = *vp;
    uu = rho * uu + gg;
    ww = ww + uu;
    *up = uu;
    *vp = ww;
  }
  if constexpr (RAGGED) {
    const int64_t i = nch * CW + sub;
    if (w0 == 0 && i < d) {
      const float* gq = g + (int64_t)(4 * h) * d + i;
      f4 gg;
      gg.x = gq[0];
      gg.y = gq[d];
      gg.z = gq[2 * d];
      gg.w = gq[3 * d];
      f4* up = reinterpret_cast<f4*>(u + i * PP) + h;
      f4* vp = reinterpret_cast<f4*>(v + i * PP) + h;
      f4 uu = *up, ww = *vp;
      uu = rho * uu + gg;
      ww = ww + uu;
      *up = uu;
      *vp = ww;
    }
  }
}

// Any P, any alignment: one lane per (coordinate, worker) for coordinates i >= i_lo.
__global__ void __launch_bounds__(kBlock) k_accumulate_il_any(const float* __restrict__ g, float* __restrict__ u,
                                                              float* __restrict__ v, int64_t d, int P, int PP,
                                                              float rho, int64_t i_lo) {
  const int64_t n = (d - i_lo) * P;
  const int64_t stride = (int64_t)gridDim.x * kBlock;
  for (int64_t e = (int64_t)blockIdx.x * kBlock + threadIdx.x; e < n; e += stride) {
    const int64_t i = i_lo + e / P;
    const int q = (int)(e % P);
    const int64_t o = i * PP + q;
    const float un = rho * u[o] + g[(int64_t)q * d + i];
    u[o] = un;
    v[o] = v[o] + un;
  }
}

__global__ void __launch_bounds__(kBlock) k_fill_zero(float* __restrict__ p, int64_t n) {
  const int64_t stride = (int64_t)gridDim.x * kBlock;
  const int64_t n4 = n / 4;
  float4* p4 = reinterpret_cast<float4*>(p);
  for (int64_t t = (int64_t)blockIdx.x * kBlock + threadIdx.x; t < n4; t += stride) p4[t] = make_float4(0.f, 0.f, 0.f, 0.f);
  const int64_t t = 4 * n4 + (int64_t)blockIdx.x * kBlock + threadIdx.x;
  if (t < n) p[t] = 0.f;
}

__global__ void __launch_bounds__(kBlock) k_fill_zero1(float* __restrict__ p, int64_t n) {
  const int64_t stride = (int64_t)gridDim.x * kBlock;
  for (int64_t t = (int64_t)blockIdx.x * kBlock + threadIdx.x; t < n; t += stride) p[t] = 0.f;
}

// ------------------------------------------------------------------------------------
// Count Sketch insertion (Sec. III-A; Alg. 1 sketch step). One lane per coordinate i: the
// r hashes of i are computed once and shared by all P workers (every worker uses the same
// hash family, which is what makes the sketches mergeable); each contribution
// s_j(i) * v[q][i] is added to acc[q][j][h_j(i)] with a device-scope fp64 atomic. Cells are
// summed in double precision and rounded once to fp32 afterwards (k_round_tables or the
// merge), so the result does not depend on the atomic order beyond fp64 rounding.

__global__ void __launch_bounds__(kBlock) k_sketch_atomic(HashSet hs, const float* __restrict__ v,
                                                          double* __restrict__ acc, int64_t d, int P, StateView sv) {
  const int64_t stride = (int64_t)gridDim.x * kBlock;
  const int64_t rc = (int64_t)hs.r * hs.c;
  for (int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x; i < d; i += stride) {
    for (int j = 0; j < hs.r; ++j) {
      uint32_t col, sflip;
      hash_ij(hs, j, (uint32_t)i, col, sflip);
      double* cell = acc + (int64_t)j * hs.c + col;
      for (int q = 0; q < P; ++q)
        unsafeAtomicAdd(cell + q * rc, (double)apply_sign(v[sv.at(q, i)], sflip));
    }
  }
}

__global__ void __launch_bounds__(kBlock) k_round_tables(const double* __restrict__ acc, float* __restrict__ tables,
                                                         int64_t n) {
  const int64_t stride = (int64_t)gridDim.x * kBlock;
  for (int64_t t = (int64_t)blockIdx.x * kBlock + threadIdx.x; t < n; t += stride) tables[t] = (float)acc[t];
}

__global__ void __launch_bounds__(kBlock) k_zero64(double* __restrict__ p, int64_t n) {
  const int64_t stride = (int64_t)gridDim.x * kBlock;
  for (int64_t t = (int64_t)blockIdx.x * kBlock + threadIdx.x; t < n; t += stride) p[t] = 0.0;
}

// ------------------------------------------------------------------------------------
// Binomial-tree merge of the P worker tables (Alg. 1 reduction loop), one lane per cell.

template <int P>
__global__ void __launch_bounds__(kBlock) k_merge(const float* __restrict__ tables, float* __restrict__ merged,
                                                  int64_t rc) {
  const int64_t stride = (int64_t)gridDim.x * kBlock;
  for (int64_t e = (int64_t)blockIdx.x * kBlock + threadIdx.x; e < rc; e += stride) {
    float x[P];
#pragma unroll
    for (int q = 0; q < P; ++q) x[q] = tables[q * rc + e];
    merged[e] = tree_sum<P>(x);
  }
}

__global__ void __launch_bounds__(kBlock) k_merge_dyn(const float* __restrict__ tables, float* __restrict__ merged,
                                                      int64_t rc, int P) {
  const int64_t stride = (int64_t)gridDim.x * kBlock;
  for (int64_t e = (int64_t)blockIdx.x * kBlock + threadIdx.x; e < rc; e += stride) {
    float x[kMaxWorkers];
    for (int q = 0; q < P; ++q) x[q] = tables[q * rc + e];
    merged[e] = tree_sum_dyn(x, P);
  }
}

// Same tree, reading the fp64 cell accumulators of gs_step: each worker's cell is rounded
// to fp32 first (its table value), then the fp32 values are summed in tree order.
template <int P>
__global__ void __launch_bounds__(kBlock) k_merge64(const double* __restrict__ acc, float* __restrict__ merged,
                                                    int64_t rc) {
  const int64_t stride = (int64_t)gridDim.x * kBlock;
  for (int64_t e = (int64_t)blockIdx.x * kBlock + threadIdx.x; e < rc; e += stride) {
    float x[P];
#pragma unroll
    for (int q = 0; q < P; ++q) x[q] = (float)acc[q * rc + e];
    merged[e] = tree_sum<P>(x);
  }
}

__global__ void __launch_bounds__(kBlock) k_merge64_dyn(const double* __restrict__ acc, float* __restrict__ merged,
                                                        int64_t rc, int P) {
  const int64_t stride = (int64_t)gridDim.x * kBlock;
  for (int64_t e = (int64_t)blockIdx.x * kBlock + threadIdx.x; e < rc; e += stride) {
    float x[kMaxWorkers];
    for (int q = 0; q < P; ++q) x[q] = (float)acc[q * rc + e];
    merged[e] = tree_sum_dyn(x, P);
  }
}

// ------------------------------------------------------------------------------------
// Exact values of the selected coordinates and their reset (Alg. 2, second round).

template <int P>
__global__ void __launch_bounds__(kBlock) k_gather_reset(const int32_t* __restrict__ idx, int64_t k,
                                                         float* __restrict__ u, float* __restrict__ v,
                                                         float* __restrict__ values, StateView sv, int reset_u) {
  const int64_t stride = (int64_t)gridDim.x * kBlock;
  for (int64_t t = (int64_t)blockIdx.x * kBlock + threadIdx.x; t < k; t += stride) {
    const int64_t i = idx[t];
    float x[P];
#pragma unroll
    for (int q = 0; q < P; ++q) x[q] = v[sv.at(q, i)];
    values[t] = tree_sum<P>(x);
#pragma unroll
    for (int q = 0; q < P; ++q) {
      v[sv.at(q, i)] = 0.f;
      if (reset_u) u[sv.at(q, i)] = 0.f;
    }
  }
}

__global__ void __launch_bounds__(kBlock) k_gather_reset_dyn(const int32_t* __restrict__ idx, int64_t k,
                                                             float* __restrict__ u, float* __restrict__ v,
                                                             float* __restrict__ values, StateView sv, int reset_u,
                                                             int P) {
  const int64_t stride = (int64_t)gridDim.x * kBlock;
  for (int64_t t = (int64_t)blockIdx.x * kBlock + threadIdx.x; t < k; t += stride) {
    const int64_t i = idx[t];
    float x[kMaxWorkers];
    for (int q = 0; q < P; ++q) x[q] = v[sv.at(q, i)];
    values[t] = tree_sum_dyn(x, P);
    for (int q = 0; q < P; ++q) {
      v[sv.at(q, i)] = 0.f;
      if (reset_u) u[sv.at(q, i)] = 0.f;
    }
  }
}

// Weight update of the selected coordinates (Alg. 1, last step): w[idx[t]] -= lr * values[t],
// the product and the difference each rounded (no fused multiply-add).
__global__ void __launch_bounds__(kBlock) k_apply_update(const int32_t* __restrict__ idx,
                                                         const float* __restrict__ values, int64_t k, float lr,
                                                         float* __restrict__ w) {
  const int64_t stride = (int64_t)gridDim.x * kBlock;
  for (int64_t t = (int64_t)blockIdx.x * kBlock + threadIdx.x; t < k; t += stride) {
    const int64_t i = idx[t];
    const float step = lr * values[t];
    w[i] = w[i] - step;
  }
}

}  // namespace

// ------------------------------------------------------------------------------------
// Launchers

namespace {
hipError_t launch_accumulate_il(const gs_ctx* x, hipStream_t s, const float* g, float* u, float* v) {
  const int P = x->P, PP = x->state_stride;
  int64_t done = 0;
  if (P % 4 == 0 && P <= 16 && aligned16(u) && aligned16(v)) {
    const int G = P / 4;
    const int64_t cw = 64 / G;
    const int64_t nch = (x->d + cw - 1) / cw;  // the last one may be ragged
    // about four chunks per wave (the most loads in flight measured best on the 25.6M x 8 stream)
    const dim3 grid(grid_for(nch, 4 * (kBlock / 64), 64 * x->num_cus)), block(kBlock);
    const bool ragged = x->d % cw != 0;
#define GS_ACC_IL(GG)                                                                               \
  if (ragged)                                                                                       \
    hipLaunchKernelGGL((k_accumulate_il<GG, true>), grid, block, 0, s, g, u, v, x->d, x->rho);      \
  else                                                                                              \
    hipLaunchKernelGGL((k_accumulate_il<GG, false>), grid, block, 0, s, g, u, v, x->d, x->rho)
    switch (G) {
      case 1: GS_ACC_IL(1); break;
      case 2: GS_ACC_IL(2); break;
      case 3: GS_ACC_IL(3); break;
      default: GS_ACC_IL(4); break;
    }
#undef GS_ACC_IL
    done = x->d;
  }
  if (done < x->d) {
    const int64_t n = (x->d - done) * P;
    hipLaunchKernelGGL(k_accumulate_il_any, dim3(grid_for(n, kBlock, 8 * x->num_cus)), dim3(kBlock), 0, s, g, u, v,
                       x->d, P, PP, x->rho, done);
  }
  return hipGetLastError();
}
}  // namespace

hipError_t launch_accumulate(const gs_ctx* x, hipStream_t s, const float* g, float* u, float* v) {
  if (x->state_layout == GS_STATE_INTERLEAVED) return launch_accumulate_il(x, s, g, u, v);
  const int64_t n = (int64_t)x->P * x->d;
  if (aligned16(g) && aligned16(u) && aligned16(v)) {
    const int64_t n4 = n / 4;
    if (n4 > 0) {
      // one group of four 64-quad chunks per wave and pass, up to 64 workgroups per CU
      const int64_t groups = n4 / (64 * 4);
      const int blocks = grid_for(groups > 0 ? groups : 1, kBlock / 64, 64 * x->num_cus);
      hipLaunchKernelGGL(k_accumulate4, dim3(blocks), dim3(kBlock), 0, s, reinterpret_cast<const f4*>(g),
                         reinterpret_cast<f4*>(u), reinterpret_cast<f4*>(v), n4, x->rho);
    }
    if (4 * n4 < n) hipLaunchKernelGGL(k_accumulate1, dim3(1), dim3(kBlock), 0, s, g, u, v, 4 * n4, n, x->rho);
  } else {
    hipLaunchKernelGGL(k_accumulate1, dim3(grid_for(n, kBlock, 8 * x->num_cus)), dim3(kBlock), 0, s, g, u, v,
                       (int64_t)0, n, x->rho);
  }
  return hipGetLastError();
}

hipError_t launch_fill_zero(hipStream_t s, float* p, int64_t n) {
  if (n <= 0) return hipSuccess;
  if (aligned16(p))
    hipLaunchKernelGGL(k_fill_zero, dim3(grid_for(n / 4 + 1, kBlock, 2048)), dim3(kBlock), 0, s, p, n);
  else
    hipLaunchKernelGGL(k_fill_zero1, dim3(grid_for(n, kBlock, 2048)), dim3(kBlock), 0, s, p, n);
  return hipGetLastError();
}

hipError_t launch_sketch_acc(const gs_ctx* x, hipStream_t s, const float* v, StateView sv) {
  const int64_t n = (int64_t)x->P * x->r * x->c;
  hipLaunchKernelGGL(k_zero64, dim3(grid_for(n, kBlock, 2048)), dim3(kBlock), 0, s, x->acc64, n);
  hipLaunchKernelGGL(k_sketch_atomic, dim3(grid_for(x->d, kBlock, 8 * x->num_cus)), dim3(kBlock), 0, s, x->hs, v,
                     x->acc64, x->d, x->P, sv);
  return hipGetLastError();
}

hipError_t launch_sketch(const gs_ctx* x, hipStream_t s, const float* v, StateView sv, float* tables) {
  hipError_t e = launch_sketch_acc(x, s, v, sv);
  if (e != hipSuccess) return e;
  const int64_t n = (int64_t)x->P * x->r * x->c;
  hipLaunchKernelGGL(k_round_tables, dim3(grid_for(n, kBlock, 2048)), dim3(kBlock), 0, s, x->acc64, tables, n);
  return hipGetLastError();
}

hipError_t launch_merge(const gs_ctx* x, hipStream_t s, const float* tables, float* merged) {
  const int64_t rc = (int64_t)x->r * x->c;
  const dim3 grid(grid_for(rc, kBlock, 8 * x->num_cus)), block(kBlock);
  switch (x->P) {
#define GS_MERGE_CASE(PP) \
  case PP: hipLaunchKernelGGL(k_merge<PP>, grid, block, 0, s, tables, merged, rc); break;
    GS_MERGE_CASE(1) GS_MERGE_CASE(2) GS_MERGE_CASE(3) GS_MERGE_CASE(4) GS_MERGE_CASE(5) GS_MERGE_CASE(6)
    GS_MERGE_CASE(7) GS_MERGE_CASE(8) GS_MERGE_CASE(9) GS_MERGE_CASE(10) GS_MERGE_CASE(11) GS_MERGE_CASE(12)
    GS_MERGE_CASE(13) GS_MERGE_CASE(14) GS_MERGE_CASE(15) GS_MERGE_CASE(16)
#undef GS_MERGE_CASE
    default: hipLaunchKernelGGL(k_merge_dyn, grid, block, 0, s, tables, merged, rc, x->P); break;
  }
  return hipGetLastError();
}

hipError_t launch_merge_acc(const gs_ctx* x, hipStream_t s, float* merged) {
  const int64_t rc = (int64_t)x->r * x->c;
  const dim3 grid(grid_for(rc, kBlock, 8 * x->num_cus)), block(kBlock);
  switch (x->P) {
#define GS_MERGE_CASE(PP) \
  case PP: hipLaunchKernelGGL(k_merge64<PP>, grid, block, 0, s, x->acc64, merged, rc); break;
    GS_MERGE_CASE(1) GS_MERGE_CASE(2) GS_MERGE_CASE(3) GS_MERGE_CASE(4) GS_MERGE_CASE(5) GS_MERGE_CASE(6)
    GS_MERGE_CASE(7) GS_MERGE_CASE(8) GS_MERGE_CASE(9) GS_MERGE_CASE(10) GS_MERGE_CASE(11) GS_MERGE_CASE(12)
    GS_MERGE_CASE(13) GS_MERGE_CASE(14) GS_MERGE_CASE(15) GS_MERGE_CASE(16)
#undef GS_MERGE_CASE
    default: hipLaunchKernelGGL(k_merge64_dyn, grid, block, 0, s, x->acc64, merged, rc, x->P); break;
  }
  return hipGetLastError();
}

hipError_t launch_gather_reset(const gs_ctx* x, hipStream_t s, const int32_t* idx, int64_t k, float* u, float* v,
                               float* values) {
  const dim3 grid(grid_for(k, kBlock, 4 * x->num_cus)), block(kBlock);
  const int ru = x->reset_momentum ? 1 : 0;
  const StateView sv = state_view(x);
  switch (x->P) {
#define GS_GATHER_CASE(PP) \
  case PP: hipLaunchKernelGGL(k_gather_reset<PP>, grid, block, 0, s, idx, k, u, v, values, sv, ru); break;
    GS_GATHER_CASE(1) GS_GATHER_CASE(2) GS_GATHER_CASE(3) GS_GATHER_CASE(4) GS_GATHER_CASE(5) GS_GATHER_CASE(6)
    GS_GATHER_CASE(7) GS_GATHER_CASE(8) GS_GATHER_CASE(9) GS_GATHER_CASE(10) GS_GATHER_CASE(11) GS_GATHER_CASE(12)
    GS_GATHER_CASE(13) GS_GATHER_CASE(14) GS_GATHER_CASE(15) GS_GATHER_CASE(16)
#undef GS_GATHER_CASE
    default: hipLaunchKernelGGL(k_gather_reset_dyn, grid, block, 0, s, idx, k, u, v, values, sv, ru, x->P); break;
  }
  return hipGetLastError();
}

hipError_t launch_apply_update(const gs_ctx* x, hipStream_t s, const int32_t* idx, const float* values, int64_t k,
                               float lr, float* w) {
  hipLaunchKernelGGL(k_apply_update, dim3(grid_for(k, kBlock, 4 * x->num_cus)), dim3(kBlock), 0, s, idx, values, k, lr,
                     w);
  return hipGetLastError();
}

}  // namespace gs
