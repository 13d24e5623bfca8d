// k_pull.hip -- Count Sketch insertion as a gather ("pull") into LDS-resident tiles.
//
// The sketch S^q[j][col] = sum over {i : h_j(i) = col} of s_j(i) v^q_i (Sec. III-A) is
// computed per column tile instead of by scattering: a tile is a range of W columns of one
// row j, held for all P workers in LDS as fp64 accumulators. Because the hash family is
// fixed for the life of a context, the set of coordinates that land in each tile is fixed
// too; gs_create builds it once as per-tile coordinate lists in ascending order (three
// passes: per-chunk counts, offsets, an in-order fill). Each step then
//   1. accumulates (u, v) and writes v worker-interleaved, vI[i][q] (one contiguous row of
//      P floats per coordinate), so one gather serves every worker;
//   2. runs one workgroup per (tile, list segment): gather vI rows of the listed
//      coordinates, add s_j(i) * vI[i][q] into the LDS tile (worker-major, fp64, LDS
//      atomics) and write the tile out (no global atomics);
//   3. sums the segments of each cell in fixed order (fp64), rounds once to fp32 (the
//      worker's table value) and merges the workers in the binomial-tree order.
// All tiles walk their lists in ascending coordinate order at similar rates, so at any
// moment the gathers of all tiles fall in a narrow band of vI that stays in cache.
#include <system_error>
#include <thread>
#include <type_traits>
#include <vector>

#include "gs_internal.hpp"

namespace gs {
namespace {

constexpr int kBlock = 256;
// Threads of a pull workgroup (one tile per CU, see make_pull_plan) and list entries in
// flight per lane group. The pull waits on L2 requests (each CU keeps a bounded number in
// flight, and most first touches of a line miss), so it wants many gathers outstanding:
// measured best at 512 threads and about 1,500 entries per CU (4 per group when one lane
// takes an entry, P <= 4; 6 otherwise).
constexpr int kPullBlock = 512;
constexpr int pull_unroll(int P) { return P <= 4 ? 4 : 6; }
// Whether a pass fetches the next pass's list words while its own rows are in flight (see
// k_pull): the one-worker plain-vector gather and four lanes per entry (P >= 13).
constexpr bool pull_pipelined(int P, bool flat) { return flat || P >= 13; }
typedef float f4 __attribute__((ext_vector_type(4)));

int grid_for(int64_t work_items, int per_block, int cap) {
  int64_t b = (work_items + per_block - 1) / per_block;
  if (b < 1) b = 1;
  if (b > cap) b = cap;
  return (int)b;
}

// theta * col mod c for theta < 2^22 and col < c < 2^31: the product is below 2^53, so it
// and its quotient estimate in double precision are within one of the true quotient.
__device__ __forceinline__ uint32_t scaled_position(uint32_t theta, uint32_t col, uint32_t c, double inv_c) {
  const uint64_t prod = (uint64_t)theta * col;
  const uint64_t q = (uint64_t)((double)prod * inv_c);
  int64_t rem = (int64_t)(prod - q * (uint64_t)c);
  if (rem < 0) rem += c;
  if (rem >= (int64_t)c) rem -= c;
  return (uint32_t)rem;
}

// The tile of entry (j, i) and the entry's position in it (the scaled column t = theta_j *
// col mod c, less the tile's first position), and the sign as a float sign-bit mask.
__device__ __forceinline__ void tile_of(const HashSet& hs, const PullPlan& pl, int j, uint32_t i, uint32_t& pos,
                                        uint32_t& sflip, uint32_t& tile) {
  uint32_t col;
  hash_ij(hs, j, i, col, sflip);
  const uint32_t t = scaled_position(pl.theta[j], col, hs.c, pl.inv_c);
  const uint32_t k = (uint32_t)(((uint64_t)t * pl.w_magic) >> pl.w_shift);  // t / W
  tile = (uint32_t)j * pl.tiles_per_row + k;
  pos = t - k * (uint32_t)pl.W;
}

// Lanes of the wave whose `t` equals this lane's (t < 2^nbits), by one ballot per bit.
__device__ __forceinline__ uint64_t same_value_lanes(uint32_t t, bool valid, int nbits) {
  uint64_t m = __ballot(valid);
  for (int b = 0; b < nbits; ++b) {
    const bool bit = (t >> b) & 1u;
    const uint64_t ones = __ballot(valid && bit);
    m &= bit ? ones : ~ones;
  }
  return m;
}

// Work item of pull workgroup b (of n): the workgroups of one round (`slots` resident at a
// time, one per CU) are dealt to the 8 XCDs in turn (b mod 8), so each XCD is given a
// contiguous run of the round's items, i.e. neighbouring tiles of one row. A 128-byte line
// of the state then feeds one XCD per row instead of one per tile it touches.
__device__ __forceinline__ int64_t grouped_item(int64_t b, int64_t n, int64_t slots) {
  const int64_t r0 = (b / slots) * slots;
  const int64_t nr = min(slots, n - r0);
  const int64_t w = b - r0, x = w % 8, q = nr / 8, rem = nr % 8;
  return r0 + x * q + min(x, rem) + w / 8;
}

// Column of position `pos` of tile k of row j (the inverse scaling).
__device__ __forceinline__ uint32_t column_at(const HashSet& hs, const PullPlan& pl, int j, int64_t k, int64_t pos) {
  return (uint32_t)(((uint64_t)pl.theta_inv[j] * (uint64_t)(k * pl.W + pos)) % hs.c);
}

// LDS cell of tile position t. A row whose common step between consecutive coordinates is a
// multiple of 2^s would put a run's cells t, t + step, ... in 32 / 2^s of the 32 bank pairs
// of fp64 cells; XOR-ing the low five bits with bits s .. s + 4 (which advance by an odd
// amount each step) spreads them over all. Only the low five bits change, bit i by bit i + s,
// so the map is a bijection on every aligned block of 32 cells.
__device__ __forceinline__ uint32_t tile_cell(uint32_t t, int swz) {
  return swz ? t ^ ((t >> swz) & 31u) : t;
}

// ------------------------------------------------------------------------------------
// Static list build (gs_create).

// counts[b][t]: entries of build chunk b that fall in tile t (every t written). The chunk's
// counts are an LDS histogram; consecutive coordinates mostly share a tile, so the lanes of
// a wave add per distinct tile, once (a ballot per tile).
__global__ void __launch_bounds__(kBlock) k_build_count(HashSet hs, PullPlan pl, int64_t d,
                                                        uint32_t* __restrict__ counts) {
  extern __shared__ uint32_t h[];  // [T]
  const int64_t b = blockIdx.x;
  for (int64_t t = threadIdx.x; t < pl.T; t += kBlock) h[t] = 0u;
  __syncthreads();
  const int lane = threadIdx.x & 63;
  const uint64_t below = (1ull << lane) - 1ull;
  const int64_t lo = b * pl.chunk, hi = min(d, lo + pl.chunk);
  for (int64_t i0 = lo; i0 < hi; i0 += kBlock) {  // block-uniform
    const int64_t i = i0 + threadIdx.x;
    const bool valid = i < hi;
    for (int j = 0; j < hs.r; ++j) {
      uint32_t pos = 0, sflip = 0, t = 0;
      if (valid) tile_of(hs, pl, j, (uint32_t)i, pos, sflip, t);
      // the first lane of each distinct tile adds the tile's lane count (distinct addresses)
      const uint64_t same = same_value_lanes(t, valid, pl.tile_bits);
      if (valid && (same & below) == 0ull) atomicAdd(&h[t], (uint32_t)__popcll(same));
    }
  }
  __syncthreads();
  for (int64_t t = threadIdx.x; t < pl.T; t += kBlock) counts[b * pl.T + t] = h[t];
}

// Per tile: exclusive prefix of counts over chunks (in place) and the tile total.
__global__ void __launch_bounds__(kBlock) k_build_prefix(PullPlan pl, uint32_t* __restrict__ counts,
                                                         uint32_t* __restrict__ total) {
  const int64_t t = (int64_t)blockIdx.x * kBlock + threadIdx.x;
  if (t >= pl.T) return;
  uint32_t run = 0;
#pragma unroll 8
  for (int64_t b = 0; b < pl.NB; ++b) {
    const uint32_t cnt = counts[b * pl.T + t];
    counts[b * pl.T + t] = run;
    run += cnt;
  }
  total[t] = run;
}

// Tile start offsets by one block: each tile's list starts at a multiple of kListGroup
// (exclusive scan of the totals rounded up); off[T] is the padded length. n[t] = total[t].
__global__ void __launch_bounds__(1024) k_build_offsets(PullPlan pl, const uint32_t* __restrict__ total,
                                                        int64_t* __restrict__ off, uint32_t* __restrict__ n) {
  __shared__ int64_t part[1024];
  const int64_t per = (pl.T + 1023) / 1024;
  const int64_t lo = threadIdx.x * per, hi = min((int64_t)pl.T, lo + per);
  auto padded = [](uint32_t x) { return ((int64_t)x + kListGroup - 1) / kListGroup * kListGroup; };
  int64_t s = 0;
  for (int64_t t = lo; t < hi; ++t) s += padded(total[t]);
  part[threadIdx.x] = s;
  __syncthreads();
  if (threadIdx.x == 0) {
    int64_t run = 0;
    for (int w = 0; w < 1024; ++w) {
      const int64_t x = part[w];
      part[w] = run;
      run += x;
    }
    off[pl.T] = run;
  }
  __syncthreads();
  int64_t run = part[threadIdx.x];
  for (int64_t t = lo; t < hi; ++t) {
    off[t] = run;
    n[t] = total[t];
    run += padded(total[t]);
  }
}

// Group bases of the packed lists: the first coordinate of each group of kListGroup entries
// (every group holds at least one entry of its tile: tiles start at group boundaries).
__global__ void __launch_bounds__(kBlock) k_build_bases(const uint32_t* __restrict__ list, int64_t groups,
                                                        uint32_t* __restrict__ bases) {
  const int64_t stride = (int64_t)gridDim.x * kBlock;
  for (int64_t g = (int64_t)blockIdx.x * kBlock + threadIdx.x; g < groups; g += stride)
    bases[g] = list[g * kListGroup];
}

// One block per tile: does every entry's offset from its group base fit in off_bits bits?
// (flag set otherwise). With pack = 1, rewrite the entries in place as packed words.
__global__ void __launch_bounds__(kBlock) k_build_pack(uint32_t* __restrict__ list, const uint16_t* __restrict__ codes,
                                                       const uint32_t* __restrict__ bases,
                                                       const int64_t* __restrict__ off,
                                                       const uint32_t* __restrict__ n, int off_bits, int pack,
                                                       uint32_t* __restrict__ flag) {
  const int64_t t = blockIdx.x;
  const int64_t lo = off[t], hi = lo + n[t];
  const uint32_t lim = 1u << off_bits;
  bool bad = false;
  for (int64_t e = lo + threadIdx.x; e < hi; e += kBlock) {
    const uint32_t o = list[e] - bases[e / kListGroup];  // entries ascend within a tile
    if (o >= lim) bad = true;
    if (pack) {
      const uint32_t code = codes[e];
      list[e] = o | ((code & 0x7fffu) << off_bits) | ((code & 0x8000u) << 16);
    }
  }
  if (bad) atomicOr(flag, 1u);
}

// In-order fill: one wave per build chunk walks its coordinates in ascending order, 64 at
// a time (lane order = coordinate order). The lanes whose entry falls in one tile take
// consecutive slots in lane order: per distinct tile of the wave, its first lane advances
// the tile's cursor by the number of such lanes and each lane adds its rank among them. So
// every tile's list comes out sorted by coordinate.
__global__ void __launch_bounds__(64) k_build_fill(HashSet hs, PullPlan pl, int64_t d,
                                                   const uint32_t* __restrict__ prefix,
                                                   const int64_t* __restrict__ off, uint32_t* __restrict__ list,
                                                   uint16_t* __restrict__ codes) {
  extern __shared__ uint32_t cursor[];  // [T]
  const int64_t b = blockIdx.x;
  const int lane = threadIdx.x;
  for (int64_t t = lane; t < pl.T; t += 64) cursor[t] = prefix[b * pl.T + t];
  __syncthreads();
  const uint64_t below = (1ull << lane) - 1ull;
  const int64_t lo = b * pl.chunk, hi = min(d, lo + pl.chunk);
  for (int64_t base = lo; base < hi; base += 64) {
    const int64_t i = base + lane;
    const bool valid = i < hi;
    for (int j = 0; j < hs.r; ++j) {
      uint32_t pos = 0, sflip = 0, t = 0;
      if (valid) tile_of(hs, pl, j, (uint32_t)i, pos, sflip, t);
      // per distinct tile, its first lane advances the cursor by the tile's lane count (the
      // leaders hold distinct tiles, so their reads and writes do not collide) and every lane
      // adds its rank among the tile's lanes
      const uint64_t same = same_value_lanes(t, valid, pl.tile_bits);
      const int leader = same ? __builtin_ctzll(same) : lane;
      uint32_t start = 0;
      if (valid && leader == lane) {
        start = cursor[t];
        cursor[t] = start + (uint32_t)__popcll(same);
      }
      start = __shfl(start, leader, 64);
      const uint32_t slot = start + (uint32_t)__popcll(same & below);
      if (valid) {
        list[off[t] + slot] = (uint32_t)i;
        codes[off[t] + slot] = (uint16_t)(pos | (sflip >> 16));  // position < 2^15; sign in bit 15
      }
    }
  }
}

// ------------------------------------------------------------------------------------
// Per step: accumulation that also writes the worker-interleaved copy of v.
// One lane handles 4 consecutive coordinates of every worker (float4 per worker row).

// Worker-major arrays ([P][d]) into the interleaved copy vI ([d][PP] rows, PP = P rounded up
// to 4), with (ACC) or without the accumulation of u and v on the way. A wave covers CW =
// 64/G consecutive coordinates, G = PP/4 16-byte pieces per row: lane l takes coordinate
// l/G and piece h = l%G (workers 4h .. 4h+3). So the worker-major loads and stores are 4
// bytes per lane and 4*CW contiguous bytes per worker row and instruction, and the vI
// stores 16 bytes per lane, 16*CW*G contiguous bytes per instruction. Each pass a wave takes
// U consecutive chunks (U below), all in flight together; the chunks past the last such
// group, the ragged last one included (lanes past d take no coordinate), run one at a time.
// Workers past P read nothing and write 0 into vI.
template <int P, bool ACC>
__global__ void __launch_bounds__(kBlock) k_vi_il(const float* __restrict__ g, float* __restrict__ u,
                                                  float* __restrict__ v, float* __restrict__ vI, int64_t d,
                                                  float rho) {
  constexpr int PP = (P + 3) & ~3;
  constexpr int G = PP / 4;
  constexpr int CW = 64 / G;
  // chunks per wave and pass: eight with the accumulation for P > 4 (worker-major step at
  // d = 25.6M x 8: 0.947 -> 0.916 ms with the scheduling barrier below, 66M x 16: 6.61 ->
  // 5.90 ms), else four (the interleave alone, and P <= 4, measured no better with eight)
  constexpr int U = ACC && P > 4 ? 8 : 4;
  const int lane = threadIdx.x & 63;
  if (lane >= CW * G) return;  // G = 3: one idle lane per wave (no barrier below)
  const int h = lane % G;
  const int64_t sub = lane / G;
  const int64_t nch = (d + CW - 1) / CW;
  const int64_t ngr = (d / CW) / U;  // groups of U full chunks
  const int64_t wstride = (int64_t)gridDim.x * (kBlock / 64);
  const int64_t w0 = (int64_t)blockIdx.x * (kBlock / 64) + (threadIdx.x >> 6);
  // one pass over n consecutive chunks starting at chunk c0 (this lane's coordinate in each)
  auto pass = [&](int64_t c0, auto n_const) {
    constexpr int N = decltype(n_const)::value;
    float x[N][4], uu[N][4], gg[N][4];
#pragma unroll
    for (int m = 0; m < N; ++m) {
      const int64_t i = (c0 + m) * CW + sub;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int w = 4 * h + q;
        x[m][q] = 0.f;
        uu[m][q] = 0.f;
        gg[m][q] = 0.f;
        if (w < P) {
          const int64_t o = (int64_t)w * d + i;
          if constexpr (ACC) {
            gg[m][q] = __builtin_nontemporal_load(g + o);
            uu[m][q] = __builtin_nontemporal_load(u + o);
          }
          x[m][q] = __builtin_nontemporal_load(v + o);
        }
      }
    }
    // P = 5..8: every load of the pass issued before any arithmetic (measured faster there,
    // slower for P = 16)
    if constexpr (ACC && P > 4 && P <= 8) __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int m = 0; m < N; ++m) {
      const int64_t i = (c0 + m) * CW + sub;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int w = 4 * h + q;
        if (ACC && w < P) {
          const int64_t o = (int64_t)w * d + i;
          uu[m][q] = rho * uu[m][q] + gg[m][q];
          x[m][q] = x[m][q] + uu[m][q];
          __builtin_nontemporal_store(uu[m][q], u + o);
          __builtin_nontemporal_store(x[m][q], v + o);
        }
      }
      f4 row;
      row.x = x[m][0];
      row.y = x[m][1];
      row.z = x[m][2];
      row.w = x[m][3];
      reinterpret_cast<f4*>(vI + i * PP)[h] = row;
    }
  };
  for (int64_t gr = w0; gr < ngr; gr += wstride) pass(gr * U, std::integral_constant<int, U>());
  for (int64_t ch = ngr * U + w0; ch < nch; ch += wstride)
    if (ch * CW + sub < d) pass(ch, std::integral_constant<int, 1>());
}

// Generic (any P, any d, any alignment): one lane per (coordinate, worker).
// Coordinates from i_lo on.
__global__ void __launch_bounds__(kBlock) k_accumulate_vi_any(const float* __restrict__ g, float* __restrict__ u,
                                                              float* __restrict__ v, float* __restrict__ vI,
                                                              int64_t d, int P, int PP, float rho, int do_acc,
                                                              int64_t i_lo) {
  const int64_t dt = d - i_lo;
  const int64_t n = (int64_t)P * dt;
  const int64_t stride = (int64_t)gridDim.x * kBlock;
  for (int64_t t = (int64_t)blockIdx.x * kBlock + threadIdx.x; t < n; t += stride) {
    const int64_t q = t / dt, i = i_lo + (t - q * dt);
    const int64_t e = q * d + i;
    float w;
    if (do_acc) {
      const float un = rho * u[e] + g[e];
      u[e] = un;
      w = v[e] + un;
      v[e] = w;
    } else {
      w = v[e];
    }
    vI[i * PP + q] = w;
  }
}

// Copy of an interleaved state array that is not 16-byte aligned (any alignment, one float
// per lane), so that the pull can load 16-byte pieces of its rows.
__global__ void __launch_bounds__(kBlock) k_copy_rows(const float* __restrict__ src, float* __restrict__ dst,
                                                      int64_t n) {
  const int64_t stride = (int64_t)gridDim.x * kBlock;
  for (int64_t e = (int64_t)blockIdx.x * kBlock + threadIdx.x; e < n; e += stride) dst[e] = src[e];
}

// ------------------------------------------------------------------------------------
// The pull: one workgroup per (tile, segment).

template <int PP>
__device__ __forceinline__ void load_row(const float* __restrict__ vI, uint32_t i, float (&x)[PP]) {
  const f4* p = reinterpret_cast<const f4*>(vI + (int64_t)i * PP);
#pragma unroll
  for (int m = 0; m < PP / 4; ++m) {
    const f4 y = p[m];
    x[4 * m + 0] = y.x;
    x[4 * m + 1] = y.y;
    x[4 * m + 2] = y.z;
    x[4 * m + 3] = y.w;
  }
}

// L = PP/4 adjacent lanes share one list entry; lane `sub` of the group gathers workers
// [4 sub, 4 sub + 4) of the row (16 B) and adds them into the tile.
// With one list segment per tile (S = 1) the tile holds every worker's complete fp64 cell
// sums, so it rounds them itself: tables[q] (when non-null) and the tree-order merge into
// `merged` (when non-null) are written directly, and the fp64 partials are not. Otherwise
// (S > 1, or both outputs null) the partials go to `partial` for k_merge_partials.
// List entry e: its coordinate i, position in the tile and sign mask (from a packed word and
// its group base, or from the unpacked list and codes).
template <bool PK>
__device__ __forceinline__ void decode_entry(uint32_t w, uint32_t aux, int off_bits, uint32_t& i, uint32_t& pos,
                                             uint32_t& sflip) {
  if constexpr (PK) {
    i = aux + (w & ((1u << off_bits) - 1u));
    pos = (w & 0x7fffffffu) >> off_bits;
    sflip = w & 0x80000000u;
  } else {
    i = w;
    pos = aux & 0x7fffu;
    sflip = (aux & 0x8000u) << 16;
  }
}

// Segment s of the S segments of a tile's list [lo, lo + n): inner boundaries are rounded
// down to multiples of kListGroup entries from lo, which is itself such a multiple, so a
// segment never splits a group of the packed list.
__device__ __forceinline__ void segment_bounds(int64_t lo, int64_t n, int64_t s, int64_t S, int64_t& e0,
                                               int64_t& e1) {
  constexpr int64_t g = kListGroup;
  e0 = lo + (n * s / S) / g * g;
  e1 = s + 1 == S ? lo + n : lo + (n * (s + 1) / S) / g * g;
}

// Workers 4 sub .. 4 sub + 3 of coordinate i: one 16-byte load of an interleaved row (rows of
// PP floats, 16-byte aligned), or, with FLAT (one worker: the state [1][d] is a plain vector),
// the coordinate's one value.
template <int P, bool FLAT>
__device__ __forceinline__ f4 load_quad(const float* __restrict__ v, uint32_t i, int sub) {
  constexpr int PP = (P + 3) & ~3;
  if constexpr (FLAT) {
    static_assert(P == 1, "a flat state holds one worker");
    f4 x;
    x.x = v[i];
    x.y = x.z = x.w = 0.f;
    return x;
  } else {
    return reinterpret_cast<const f4*>(v + (int64_t)i * PP)[sub];
  }
}

template <int P, int U, bool PK, bool FLAT>
__global__ void __launch_bounds__(kPullBlock) k_pull(HashSet hs, PullPlan pl, const uint32_t* __restrict__ list,
                                                     const uint16_t* __restrict__ codes,
                                                     const uint32_t* __restrict__ bases,
                                                     const int64_t* __restrict__ off, const uint32_t* __restrict__ tn,
                                                     const float* __restrict__ vI, double* __restrict__ partial,
                                                     float* __restrict__ merged, float* __restrict__ tables) {
  extern __shared__ double acc[];  // [P][ws] (below): worker-major, so lanes adding for one worker hit spread banks
  constexpr int PP = (P + 3) & ~3;
  constexpr int L = PP / 4;
  constexpr int64_t B = kPullBlock / L;  // entries per block pass
  const int sub = threadIdx.x % L;
  // Lane group tid0 takes list entry tid (of each block pass). Consecutive entries of a tile
  // are mostly consecutive coordinates at scaled positions t, t + s, t + 2s, ..., and with two
  // lanes per entry (P = 5..8) such runs on neighbouring lanes made the LDS atomics conflict:
  // permuting the entries within each aligned group of 32 (the entries one wave instruction
  // covers, so the L2 requests are unchanged) took the pull from 0.885 to 0.739 ms at
  // d = 25.6M x 8. With one or four lanes per entry the same permutation measured slower.
  const int64_t tid0 = threadIdx.x / L;
  const int64_t tid = (L == 2 && (tid0 | 31) < B) ? ((tid0 & ~31ll) | ((tid0 * 13 + 7) & 31)) : tid0;
  const int64_t item = grouped_item(blockIdx.x, gridDim.x, pl.slots);
  const int64_t t = item / pl.S, s = item - t * pl.S;
  const int j = (int)(t / pl.tiles_per_row);
  const int64_t kt = t - (int64_t)j * pl.tiles_per_row;
  const int64_t wt = min((int64_t)pl.W, (int64_t)hs.c - kt * pl.W);
  // column stride: whole blocks of 32 cells (for the swizzle) plus 6, so that the two or four
  // workers' columns one wave instruction adds into start in different banks
  const int64_t ws = ((wt + 31) & ~31ll) + 6;
  const int swz = pl.swz[j];
  for (int64_t e = threadIdx.x; e < ws * P; e += kPullBlock) acc[e] = 0.0;
  __syncthreads();
  int64_t e0, e1;
  segment_bounds(off[t], tn[t], s, pl.S, e0, e1);
  double* const mycol = acc + (int64_t)(4 * sub) * ws;
  // when L does not divide the block (L = 3: 85 groups of 3 lanes), the last lane has no
  // group: it takes no entry (its would be the next pass's first)
  int64_t eb = tid0 < B ? e0 + tid : e1;
  // The list words of a pass's U entries (and their group bases). Pipelined (PIPE), a pass
  // fetches the next pass's words while its own rows are in flight, so it waits on one memory
  // round trip (the rows), not two (words, then rows): measured faster where a pass moves
  // little (one worker's 4-byte values: 0.39 -> 0.30 ms at d = 25.6M) or where the miss
  // latency is long (66M x 16: 6.10 -> 5.71 ms), slower at 25.6M x 8 (0.66 -> 0.73 ms).
  constexpr bool PIPE = pull_pipelined(P, FLAT);
  uint32_t wn[U], an[U];
  auto fetch = [&](int64_t ebx) {
#pragma unroll
    for (int m = 0; m < U; ++m) {
      const int64_t e = ebx + m * B;
      wn[m] = list[e];
      if constexpr (PK && (L == 1 || L == 2 || L == 4)) {
        static_assert(B % kListGroup == 0 && kListGroup % (64 / L) == 0, "a wave's entries must share a group");
        // e0 is group-aligned, B is a multiple of kListGroup and a wave's lanes take 64 / L
        // consecutive entries of an aligned run (permuted within it): every lane active in
        // this pass needs the same group base, so the wave loads it once, as a scalar. The
        // tail loop below cannot do this (its lanes may be one pass apart).
        an[m] = bases[__builtin_amdgcn_readfirstlane((uint32_t)(e / kListGroup))];
      } else {
        an[m] = PK ? bases[e / kListGroup] : (uint32_t)codes[e];
      }
    }
  };
  if (PIPE && eb + (U - 1) * B < e1) {
    fetch(eb);
    for (;;) {
      uint32_t i[U], pos[U], sg[U];
#pragma unroll
      for (int m = 0; m < U; ++m) decode_entry<PK>(wn[m], an[m], pl.off_bits, i[m], pos[m], sg[m]);
      f4 x[U];
#pragma unroll
      for (int m = 0; m < U; ++m) x[m] = load_quad<P, FLAT>(vI, i[m], sub);
      const int64_t ebn = eb + U * B;
      const bool more = ebn + (U - 1) * B < e1;
      if (more) fetch(ebn);
#pragma unroll
      for (int m = 0; m < U; ++m) {
        double* cell = mycol + tile_cell(pos[m], swz);
        const uint32_t sflip = sg[m];
        const float xs[4] = {x[m].x, x[m].y, x[m].z, x[m].w};
#pragma unroll
        for (int q = 0; q < 4; ++q)
          if (P % 4 == 0 || 4 * sub + q < P) atomicAdd(cell + q * ws, (double)apply_sign(xs[q], sflip));
      }
      eb = ebn;
      if (!more) break;
    }
  }
  for (; !PIPE && eb + (U - 1) * B < e1; eb += U * B) {
    fetch(eb);
    uint32_t i[U], pos[U], sg[U];
#pragma unroll
    for (int m = 0; m < U; ++m) decode_entry<PK>(wn[m], an[m], pl.off_bits, i[m], pos[m], sg[m]);
    f4 x[U];
#pragma unroll
    for (int m = 0; m < U; ++m) x[m] = load_quad<P, FLAT>(vI, i[m], sub);
#pragma unroll
    for (int m = 0; m < U; ++m) {
      double* cell = mycol + tile_cell(pos[m], swz);
      const uint32_t sflip = sg[m];
      const float xs[4] = {x[m].x, x[m].y, x[m].z, x[m].w};
#pragma unroll
      for (int q = 0; q < 4; ++q)
        if (P % 4 == 0 || 4 * sub + q < P) atomicAdd(cell + q * ws, (double)apply_sign(xs[q], sflip));
    }
  }
  for (; eb < e1; eb += B) {
    uint32_t i, pos, sflip;
    decode_entry<PK>(list[eb], PK ? bases[eb / kListGroup] : (uint32_t)codes[eb], pl.off_bits, i, pos, sflip);
    const f4 x = load_quad<P, FLAT>(vI, i, sub);
    double* cell = mycol + tile_cell(pos, swz);
    const float xs[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
    for (int q = 0; q < 4; ++q)
      if (P % 4 == 0 || 4 * sub + q < P) atomicAdd(cell + q * ws, (double)apply_sign(xs[q], sflip));
  }
  __syncthreads();
  // write out: tile position o holds column theta_inv_j * (kt W + o) mod c; along the
  // block-stride loop that column advances by (256 theta_inv_j) mod c
  const int64_t rc = (int64_t)hs.r * hs.c;
  const uint32_t c = hs.c;
  const uint32_t cstep = (uint32_t)(((uint64_t)pl.theta_inv[j] * kPullBlock) % c);
  uint32_t col = threadIdx.x < wt ? column_at(hs, pl, j, kt, threadIdx.x) : 0u;
  const int64_t row0 = (int64_t)j * c;
  if (pl.S == 1 && (merged || tables)) {
    for (int64_t o = threadIdx.x; o < wt; o += kPullBlock) {
      float x[P];
      const uint32_t oc = tile_cell((uint32_t)o, swz);
#pragma unroll
      for (int q = 0; q < P; ++q) x[q] = (float)acc[q * ws + oc];
      if (tables) {
#pragma unroll
        for (int q = 0; q < P; ++q) tables[q * rc + row0 + col] = x[q];
      }
      if (merged) merged[row0 + col] = tree_sum<P>(x);
      col = col + cstep >= c ? col + cstep - c : col + cstep;
    }
    return;
  }
  double* dst = partial + s * P * rc + row0;
  for (int64_t o = threadIdx.x; o < wt; o += kPullBlock) {
    const uint32_t oc = tile_cell((uint32_t)o, swz);
#pragma unroll
    for (int q = 0; q < P; ++q) dst[q * rc + col] = acc[q * ws + oc];
    col = col + cstep >= c ? col + cstep - c : col + cstep;
  }
}

// Runtime-P variant (P > 16): rows of PP floats read element by element.
__global__ void __launch_bounds__(kBlock) k_pull_any(HashSet hs, PullPlan pl, const uint32_t* __restrict__ list,
                                                     const uint16_t* __restrict__ codes,
                                                     const int64_t* __restrict__ off, const uint32_t* __restrict__ tn,
                                                     const float* __restrict__ vI, double* __restrict__ partial) {
  extern __shared__ double acc[];
  const int P = pl.P, PP = pl.PP;
  const int64_t item = grouped_item(blockIdx.x, gridDim.x, pl.slots);
  const int64_t t = item / pl.S, s = item - t * pl.S;
  const int j = (int)(t / pl.tiles_per_row);
  const int64_t kt = t - (int64_t)j * pl.tiles_per_row;
  const int64_t wt = min((int64_t)pl.W, (int64_t)hs.c - kt * pl.W);
  for (int64_t e = threadIdx.x; e < wt * P; e += kBlock) acc[e] = 0.0;
  __syncthreads();
  int64_t e0, e1;
  segment_bounds(off[t], tn[t], s, pl.S, e0, e1);
  for (int64_t e = e0 + threadIdx.x; e < e1; e += kBlock) {
    const uint32_t i = list[e], code = codes[e];
    double* cell = acc + (code & 0x7fffu);
    const uint32_t sflip = (code & 0x8000u) << 16;
    for (int q = 0; q < P; ++q) atomicAdd(cell + q * wt, (double)apply_sign(vI[(int64_t)i * PP + q], sflip));
  }
  __syncthreads();
  const int64_t rc = (int64_t)hs.r * hs.c;
  const uint32_t c = hs.c;
  const uint32_t cstep = (uint32_t)(((uint64_t)pl.theta_inv[j] * kBlock) % c);
  uint32_t col = threadIdx.x < wt ? column_at(hs, pl, j, kt, threadIdx.x) : 0u;
  double* dst = partial + s * P * rc + (int64_t)j * c;
  for (int64_t o = threadIdx.x; o < wt; o += kBlock) {
    for (int q = 0; q < P; ++q) dst[q * rc + col] = acc[q * wt + o];
    col = col + cstep >= c ? col + cstep - c : col + cstep;
  }
}

// ------------------------------------------------------------------------------------
// Segment sum + single rounding + tree merge. partial is [S][P][r][c] fp64.

// Segments are added in ascending order per worker; the P sums are independent chains and
// the segment loop is unrolled, so many loads are in flight per lane (small sketches have
// tens of segments).
template <int P>
__global__ void __launch_bounds__(kBlock) k_merge_partials(const double* __restrict__ partial, int S, int64_t rc,
                                                           float* __restrict__ merged, float* __restrict__ tables) {
  const int64_t stride = (int64_t)gridDim.x * kBlock;
  for (int64_t e = (int64_t)blockIdx.x * kBlock + threadIdx.x; e < rc; e += stride) {
    double a[P];
#pragma unroll
    for (int q = 0; q < P; ++q) a[q] = partial[q * rc + e];
    int s = 1;
    for (; s + 3 < S; s += 4) {
      double y[4][P];
#pragma unroll
      for (int m = 0; m < 4; ++m)
#pragma unroll
        for (int q = 0; q < P; ++q) y[m][q] = partial[((int64_t)(s + m) * P + q) * rc + e];
#pragma unroll
      for (int m = 0; m < 4; ++m)
#pragma unroll
        for (int q = 0; q < P; ++q) a[q] += y[m][q];
    }
    for (; s < S; ++s)
#pragma unroll
      for (int q = 0; q < P; ++q) a[q] += partial[((int64_t)s * P + q) * rc + e];
    float x[P];
#pragma unroll
    for (int q = 0; q < P; ++q) x[q] = (float)a[q];
    if (tables) {
#pragma unroll
      for (int q = 0; q < P; ++q) tables[q * rc + e] = x[q];
    }
    if (merged) merged[e] = tree_sum<P>(x);
  }
}

__global__ void __launch_bounds__(kBlock) k_merge_partials_any(const double* __restrict__ partial, int S, int64_t rc,
                                                               int P, float* __restrict__ merged,
                                                               float* __restrict__ tables) {
  const int64_t stride = (int64_t)gridDim.x * kBlock;
  for (int64_t e = (int64_t)blockIdx.x * kBlock + threadIdx.x; e < rc; e += stride) {
    float x[kMaxWorkers];
    for (int q = 0; q < P; ++q) {
      double a = partial[q * rc + e];
      for (int s = 1; s < S; ++s) a += partial[((int64_t)s * P + q) * rc + e];
      x[q] = (float)a;
      if (tables) tables[q * rc + e] = x[q];
    }
    if (merged) merged[e] = tree_sum_dyn(x, P);
  }
}

// k_vi_il over every chunk (the last one may be ragged); g and u only with ACC.
template <int P, bool ACC>
hipError_t launch_vi_il_p(const gs_ctx* x, hipStream_t s, const float* g, float* u, float* v) {
  constexpr int CW = 64 / (((P + 3) & ~3) / 4);
  const int64_t nch = (x->d + CW - 1) / CW;
  const dim3 grid(grid_for(nch, 4 * (kBlock / 64), 64 * x->num_cus)), block(kBlock);
  hipLaunchKernelGGL((k_vi_il<P, ACC>), grid, block, 0, s, g, u, v, x->vI, x->d, x->rho);
  return hipGetLastError();
}

template <int P, bool FLAT = false>
void launch_pull_p(const gs_ctx* x, hipStream_t s, const float* rows, float* merged, float* tables) {
  const PullPlan& pl = x->plan;
  const dim3 grid((unsigned)((int64_t)pl.T * pl.S)), block(kPullBlock);
  const size_t lds = (size_t)(((pl.W + 31) & ~31) + 6) * pl.P * sizeof(double);
  if (pl.packed)
    hipLaunchKernelGGL((k_pull<P, pull_unroll(P), true, FLAT>), grid, block, lds, s, x->hs, pl, x->list, x->codes,
                       x->bases, x->tile_off, x->tile_n, rows, x->partial, merged, tables);
  else
    hipLaunchKernelGGL((k_pull<P, pull_unroll(P), false, FLAT>), grid, block, lds, s, x->hs, pl, x->list, x->codes,
                       x->bases, x->tile_off, x->tile_n, rows, x->partial, merged, tables);
}

template <int P, bool FLAT = false>
hipError_t allow_pull_lds(size_t bytes) {
  const hipError_t e = hipFuncSetAttribute(reinterpret_cast<const void*>(&k_pull<P, pull_unroll(P), true, FLAT>),
                                           hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
  if (e != hipSuccess) return e;
  return hipFuncSetAttribute(reinterpret_cast<const void*>(&k_pull<P, pull_unroll(P), false, FLAT>),
                             hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
}

}  // namespace

// ------------------------------------------------------------------------------------

namespace {

// x^-1 mod m for gcd(x, m) = 1 (extended Euclid).
uint32_t inverse_mod(uint32_t x, uint32_t m) {
  if (m == 1) return 0;
  int64_t r0 = m, r1 = x, t0 = 0, t1 = 1;
  while (r1 != 0) {
    const int64_t q = r0 / r1;
    const int64_t r2 = r0 - q * r1, t2 = t0 - q * t1;
    r0 = r1;
    r1 = r2;
    t0 = t1;
    t1 = t2;
  }
  return (uint32_t)(t0 < 0 ? t0 + m : t0);
}

uint64_t gcd_u64(uint64_t a, uint64_t b) {
  while (b) {
    const uint64_t t = a % b;
    a = b;
    b = t;
  }
  return a;
}

// The column scaling of one row: with alpha = a mod c and beta = p mod c, consecutive
// coordinates' columns differ by alpha, or by alpha - beta when the raw hash wraps past p
// (a fraction f = a / p of the steps). theta (coprime to c) minimises the expected step
// (1 - f) |theta alpha|_c + f |theta (alpha - beta)|_c of the scaled position, |x|_c being the
// distance of x mod c to 0. The search runs over theta < min(c, 2^22) with adds only.
// (Minimising instead the chance that a step leaves a tile, (1 - f) min(1, d1 / W) +
// f min(1, d2 / W), measured 10% slower at d = 66M x 16 and no faster at 25.6M x 8.)
uint32_t column_scaling(uint32_t a, int64_t c) {
  if (c <= 2) return 1;
  const uint64_t cu = (uint64_t)c;
  const uint64_t alpha = a % cu, beta = (uint64_t)kMersenne % cu;
  const uint64_t step2 = (alpha + cu - beta) % cu;
  const double f = (double)a / (double)kMersenne;
  const uint64_t limit = cu < (1ull << 22) ? cu : (1ull << 22);
  uint64_t s1 = 0, s2 = 0;
  double best = 1e300;
  uint32_t best_theta = 1;
  for (uint64_t th = 1; th < limit; ++th) {
    s1 += alpha;
    if (s1 >= cu) s1 -= cu;
    s2 += step2;
    if (s2 >= cu) s2 -= cu;
    const double d1 = (double)(s1 < cu - s1 ? s1 : cu - s1);
    const double d2 = (double)(s2 < cu - s2 ? s2 : cu - s2);
    const double cost = (1.0 - f) * d1 + f * d2;
    if (cost < best && gcd_u64(th, cu) == 1) {
      best = cost;
      best_theta = (uint32_t)th;
    }
  }
  return best_theta;
}

// The LDS swizzle of a row (tile_cell). Most consecutive coordinates of the row take one
// step, theta alpha ((1 - f) of them) or theta (alpha - beta) (f of them), at distance d from
// 0 mod c. When d is a multiple of 2^s, s >= 2, a run's cells fall into 32 / 2^s or fewer of
// the 32 bank pairs (one bank at s >= 5), and XOR-ing bits s .. s + 4 of the position into its
// low five bits spreads them over all. That scrambles the other step's runs, so it is applied
// only where the common step carries at least 3/4 of the coordinates: measured with five hash
// seeds at d = 25.6M x 8 (sketch 0.66-0.94 ms before, 0.66-0.72 after; applied also where the
// common step carries only 63%, one seed went 0.68 -> 0.72 ms).
int32_t cell_swizzle(uint32_t a, int64_t c, uint32_t theta) {
  if (c <= 2) return 0;
  const uint64_t cu = (uint64_t)c;
  const uint64_t alpha = a % cu, beta = (uint64_t)kMersenne % cu;
  const double f = (double)a / (double)kMersenne;
  if ((f > 0.5 ? f : 1.0 - f) < 0.75) return 0;
  const uint64_t step = f <= 0.5 ? alpha : (alpha + cu - beta) % cu;  // the common step
  const uint64_t t = (uint64_t)theta % cu * step % cu;
  const uint64_t dist = t < cu - t ? t : cu - t;
  if (dist == 0) return 0;
  int s = 0;
  while (((dist >> s) & 1ull) == 0ull) ++s;
  return s >= 2 ? (s > 26 ? 26 : s) : 0;
}

}  // namespace

PullPlan make_pull_plan(const HashSet& hs, int64_t d, int32_t P, int32_t r, int64_t c, int num_cus) {
  PullPlan pl{};
  {
    // the rows' scalings are independent searches of up to 2^22 steps: one thread each
    // (66M x 16, r = 7: 46 -> ~8 ms of gs_create on an 8-core host)
    auto row = [&](int j) {
      pl.theta[j] = column_scaling(hs.row[j].a, c);
      pl.theta_inv[j] = inverse_mod(pl.theta[j] % (uint32_t)c, (uint32_t)c);
      pl.swz[j] = cell_swizzle(hs.row[j].a, c, pl.theta[j]);
    };
    std::vector<std::thread> pool;
    for (int j = 1; j < r; ++j) {
      try {
        pool.emplace_back(row, j);
      } catch (const std::system_error&) {  // no thread to spare: this one does the row
        row(j);
      }
    }
    row(0);
    for (std::thread& th : pool) th.join();
  }
  pl.P = P;
  pl.PP = (P + 3) & ~3;
  // Tiles hold W columns x P workers of fp64 accumulators. Up to kTilesPerCu tiles of at
  // most 160 KiB / kTilesPerCu share a CU; W is then shrunk so that the tiles fill whole
  // rounds of resident workgroups (no ragged last round), or one round as fully as it can.
  const int64_t cu_lds = 160 * 1024;
  int64_t max_w = (cu_lds / kTilesPerCu) / (8 * (int64_t)P) - 6;
  if (max_w >= 32) max_w &= ~31ll;  // a worker's column of cells is W rounded up to 32, plus 6
  int64_t W = max_w < 1 ? 1 : max_w;
  if (W > c) W = c;
  const int64_t slots = (int64_t)kTilesPerCu * num_cus;
  pl.slots = (int32_t)(slots >= 8 ? slots / 8 * 8 : 8);
  int64_t tiles = (int64_t)r * ((c + W - 1) / W);
  if (tiles > slots) {
    const int64_t rounds = (tiles + slots - 1) / slots;
    const int64_t per_row = (rounds * slots) / r;  // tiles per row that fill `rounds` rounds
    if (per_row >= 1) {
      const int64_t w2 = (c + per_row - 1) / per_row;
      if (w2 >= 1 && w2 <= W) W = w2;
    }
  } else {
    // One round: as many tiles as there are workgroup slots (as c allows), each a single list
    // segment, rather than fewer, wider tiles split into segments. Every workgroup zeroes and
    // writes out its whole tile, so narrow tiles cost less per workgroup, and with one
    // segment per tile the tiles merge their own cells (no pass over fp64 partials): 65,536 x 4
    // 0.067 -> 0.044 ms per step (5 tiles x 4 segments -> 255 tiles), 270,000 x 4 0.091 ->
    // 0.071 ms, and d = 25.6M with one worker 0.466 -> 0.430 ms (65 tiles x 3 segments at
    // first, 85 x 3 when tiles were narrowed only as far as segments of 16 Ki entries allow).
    // Segments remain for sketches too narrow to give every slot a tile (c < slots / r).
    const int64_t tpr = std::max((c + W - 1) / W, std::min(c, slots / r));
    W = (c + tpr - 1) / tpr;
  }
  pl.W = (int32_t)W;
  {
    int pos_bits = 1;  // bits of a position in the tile (< W)
    while ((1ll << pos_bits) < W) ++pos_bits;
    pl.off_bits = 31 - pos_bits;
    pl.packed = 0;  // set by build_pull_lists when every group fits
  }
  pl.tiles_per_row = (int32_t)((c + W - 1) / W);
  pl.T = r * pl.tiles_per_row;
  {
    // t / W for t < c < 2^31 by a reciprocal multiply (as the bucket modulus), c's
    // reciprocal for theta * col mod c, and the bits of a tile index
    uint32_t l = 0;
    while ((1ull << l) < (uint64_t)W) ++l;
    pl.w_shift = 31 + l;
    pl.w_magic = (uint32_t)(((1ull << (31 + l)) + (uint64_t)W - 1) / (uint64_t)W);
    pl.inv_c = 1.0 / (double)c;
    int tb = 1;
    while ((1ll << tb) < (int64_t)pl.T) ++tb;
    pl.tile_bits = tb;
  }
  // small sketches: split each tile's list into segments so every CU gets work, at most one
  // round of workgroups (T * S <= slots: a second round would hold only the leftovers)
  int64_t S = slots / pl.T;
  const int64_t per_tile = (int64_t)r * d / pl.T;
  // every segment's workgroup zeroes and writes out a whole fp64 tile however short its list,
  // so segments stay long: at least 16 Ki entries (measured best over 0.5 .. 64 Ki at
  // d = 65,536 and 270,000)
  if (S > per_tile / 16384) S = per_tile / 16384;
  if (S < 1) S = 1;
  pl.S = (int32_t)S;
  // build chunks (one fill wave each): 16 Ki coordinates, so that the fill has several waves
  // per CU, or more for large d, so that there are at most 4,096 chunks (the per-chunk
  // counts, NB * T words, stay small and the per-tile prefix over chunks short)
  int64_t chunk = 16384;
  if ((d + chunk - 1) / chunk > 4096) chunk = ((d + 4095) / 4096 + 255) / 256 * 256;
  pl.chunk = chunk;
  pl.NB = (int32_t)((d + pl.chunk - 1) / pl.chunk);
  return pl;
}

hipError_t prepare_pull_kernels(const gs_ctx* x) {
  const size_t bytes = (size_t)(((x->plan.W + 31) & ~31) + 6) * x->plan.P * sizeof(double);
  switch (x->P) {
#define GS_ALLOW_CASE(PP) \
  case PP: return allow_pull_lds<PP>(bytes);
    case 1: {
      const hipError_t e = allow_pull_lds<1, true>(bytes);
      if (e != hipSuccess) return e;
      return allow_pull_lds<1>(bytes);
    }
    GS_ALLOW_CASE(2) GS_ALLOW_CASE(3) GS_ALLOW_CASE(4) GS_ALLOW_CASE(5) GS_ALLOW_CASE(6)
    GS_ALLOW_CASE(7) GS_ALLOW_CASE(8) GS_ALLOW_CASE(9) GS_ALLOW_CASE(10) GS_ALLOW_CASE(11) GS_ALLOW_CASE(12)
    GS_ALLOW_CASE(13) GS_ALLOW_CASE(14) GS_ALLOW_CASE(15) GS_ALLOW_CASE(16)
#undef GS_ALLOW_CASE
    default:
      return hipFuncSetAttribute(reinterpret_cast<const void*>(&k_pull_any),
                                 hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes);
  }
}

hipError_t build_pull_lists(gs_ctx* x) {
  PullPlan& pl = x->plan;
  const size_t fill_lds = (size_t)pl.T * sizeof(uint32_t);
  hipError_t ea = hipFuncSetAttribute(reinterpret_cast<const void*>(&k_build_fill),
                                      hipFuncAttributeMaxDynamicSharedMemorySize, (int)fill_lds);
  if (ea == hipSuccess)
    ea = hipFuncSetAttribute(reinterpret_cast<const void*>(&k_build_count),
                             hipFuncAttributeMaxDynamicSharedMemorySize, (int)fill_lds);
  if (ea != hipSuccess) return ea;
  ea = prepare_pull_kernels(x);
  if (ea != hipSuccess) return ea;
  uint32_t* counts = nullptr;
  uint32_t* total = nullptr;
  uint32_t* flag = nullptr;
  hipError_t e = hipMalloc(reinterpret_cast<void**>(&counts), (size_t)pl.NB * pl.T * sizeof(uint32_t));
  if (e == hipSuccess) e = hipMalloc(reinterpret_cast<void**>(&total), (size_t)pl.T * sizeof(uint32_t));
  if (e == hipSuccess) e = hipMalloc(reinterpret_cast<void**>(&flag), sizeof(uint32_t));
  if (e == hipSuccess) e = hipMemset(flag, 0, sizeof(uint32_t));
  if (e == hipSuccess) {
    hipLaunchKernelGGL(k_build_count, dim3(pl.NB), dim3(kBlock), fill_lds, 0, x->hs, pl, x->d, counts);
    hipLaunchKernelGGL(k_build_prefix, dim3((pl.T + kBlock - 1) / kBlock), dim3(kBlock), 0, 0, pl, counts, total);
    hipLaunchKernelGGL(k_build_offsets, dim3(1), dim3(1024), 0, 0, pl, total, x->tile_off, x->tile_n);
    hipLaunchKernelGGL(k_build_fill, dim3(pl.NB), dim3(64), (size_t)pl.T * sizeof(uint32_t), 0, x->hs, pl, x->d,
                       counts, x->tile_off, x->list, x->codes);
    const int64_t groups = x->list_cap / kListGroup;
    hipLaunchKernelGGL(k_build_bases, dim3(grid_for(groups, kBlock, 8 * x->num_cus)), dim3(kBlock), 0, 0, x->list,
                       groups, x->bases);
    hipLaunchKernelGGL(k_build_pack, dim3(pl.T), dim3(kBlock), 0, 0, x->list, x->codes, x->bases, x->tile_off,
                       x->tile_n, pl.off_bits, 0, flag);
    e = hipGetLastError();
  }
  uint32_t overflow = 1;
  if (e == hipSuccess) e = hipMemcpy(&overflow, flag, sizeof(uint32_t), hipMemcpyDeviceToHost);
  // pack when every group's span fits (and the unrolled pulls run: P <= 16); off_bits = 0
  // keeps the lists unpacked
  if (e == hipSuccess && overflow == 0 && x->P <= 16 && pl.off_bits > 0) {
    hipLaunchKernelGGL(k_build_pack, dim3(pl.T), dim3(kBlock), 0, 0, x->list, x->codes, x->bases, x->tile_off,
                       x->tile_n, pl.off_bits, 1, flag);
    e = hipGetLastError();
    if (e == hipSuccess) e = hipDeviceSynchronize();
    if (e == hipSuccess) {
      pl.packed = 1;
      (void)hipFree(x->codes);
      x->codes = nullptr;
    }
  }
  if (e == hipSuccess) e = hipDeviceSynchronize();
  if (counts) (void)hipFree(counts);
  if (total) (void)hipFree(total);
  if (flag) (void)hipFree(flag);
  return e;
}

hipError_t launch_accumulate_vi(const gs_ctx* x, hipStream_t s, const float* g, float* u, float* v) {
  switch (x->P) {
#define GS_ACCVI_CASE(PP) \
  case PP: return launch_vi_il_p<PP, true>(x, s, g, u, v);
    GS_ACCVI_CASE(1) GS_ACCVI_CASE(2) GS_ACCVI_CASE(3) GS_ACCVI_CASE(4) GS_ACCVI_CASE(5) GS_ACCVI_CASE(6)
    GS_ACCVI_CASE(7) GS_ACCVI_CASE(8) GS_ACCVI_CASE(9) GS_ACCVI_CASE(10) GS_ACCVI_CASE(11) GS_ACCVI_CASE(12)
    GS_ACCVI_CASE(13) GS_ACCVI_CASE(14) GS_ACCVI_CASE(15) GS_ACCVI_CASE(16)
#undef GS_ACCVI_CASE
    default: break;
  }
  const int64_t n = (int64_t)x->P * x->d;
  hipLaunchKernelGGL(k_accumulate_vi_any, dim3(grid_for(n, kBlock, 8 * x->num_cus)), dim3(kBlock), 0, s, g, u, v,
                     x->vI, x->d, x->P, x->plan.PP, x->rho, 1, (int64_t)0);
  return hipGetLastError();
}

hipError_t launch_interleave(const gs_ctx* x, hipStream_t s, const float* v) {
  float* src = const_cast<float*>(v);  // read only (no accumulation)
  switch (x->P) {
#define GS_IL_CASE(PP) \
  case PP: return launch_vi_il_p<PP, false>(x, s, nullptr, nullptr, src);
    GS_IL_CASE(1) GS_IL_CASE(2) GS_IL_CASE(3) GS_IL_CASE(4) GS_IL_CASE(5) GS_IL_CASE(6) GS_IL_CASE(7) GS_IL_CASE(8)
    GS_IL_CASE(9) GS_IL_CASE(10) GS_IL_CASE(11) GS_IL_CASE(12) GS_IL_CASE(13) GS_IL_CASE(14) GS_IL_CASE(15)
    GS_IL_CASE(16)
#undef GS_IL_CASE
    default: break;
  }
  const int64_t n = (int64_t)x->P * x->d;
  hipLaunchKernelGGL(k_accumulate_vi_any, dim3(grid_for(n, kBlock, 8 * x->num_cus)), dim3(kBlock), 0, s, nullptr,
                     nullptr, src, x->vI, x->d, x->P, x->plan.PP, x->rho, 0, (int64_t)0);
  return hipGetLastError();
}

hipError_t launch_pull_flat(const gs_ctx* x, hipStream_t s, const float* v, float* merged, float* tables) {
  if (x->P != 1) return hipErrorInvalidValue;
  launch_pull_p<1, true>(x, s, v, merged, tables);
  return hipGetLastError();
}

hipError_t launch_pull(const gs_ctx* x, hipStream_t s, const float* rows, float* merged, float* tables) {
  switch (x->P) {
#define GS_PULL_CASE(PP) \
  case PP: launch_pull_p<PP>(x, s, rows, merged, tables); break;
    GS_PULL_CASE(1) GS_PULL_CASE(2) GS_PULL_CASE(3) GS_PULL_CASE(4) GS_PULL_CASE(5) GS_PULL_CASE(6) GS_PULL_CASE(7)
    GS_PULL_CASE(8) GS_PULL_CASE(9) GS_PULL_CASE(10) GS_PULL_CASE(11) GS_PULL_CASE(12) GS_PULL_CASE(13)
    GS_PULL_CASE(14) GS_PULL_CASE(15) GS_PULL_CASE(16)
#undef GS_PULL_CASE
    default: {
      const PullPlan& pl = x->plan;
      hipLaunchKernelGGL(k_pull_any, dim3((unsigned)((int64_t)pl.T * pl.S)), dim3(kBlock),
                         (size_t)pl.W * pl.P * sizeof(double), s, x->hs, pl, x->list, x->codes, x->tile_off,
                         x->tile_n, rows, x->partial);
    }
  }
  return hipGetLastError();
}

const float* pull_rows_of_state(const gs_ctx* x, hipStream_t s, const float* v, hipError_t* e) {
  // the unrolled pulls (P <= 16) load 16-byte pieces of a row; the generic one loads floats
  if (x->P > 16 || ((uintptr_t)v & 15u) == 0) {
    *e = hipSuccess;
    return v;
  }
  const int64_t n = x->d * x->plan.PP;
  hipLaunchKernelGGL(k_copy_rows, dim3(grid_for(n, kBlock, 8 * x->num_cus)), dim3(kBlock), 0, s, v, x->vI, n);
  *e = hipGetLastError();
  return x->vI;
}

bool pull_merges(const gs_ctx* x) { return x->P <= 16 && x->plan.S == 1; }

hipError_t launch_merge_partials(const gs_ctx* x, hipStream_t s, float* merged, float* tables) {
  if (pull_merges(x)) return hipSuccess;  // the pull wrote merged / tables itself
  const int64_t rc = (int64_t)x->r * x->c;
  const dim3 grid(grid_for(rc, kBlock, 8 * x->num_cus)), block(kBlock);
  const int S = x->plan.S;
  switch (x->P) {
#define GS_MP_CASE(PP) \
  case PP: hipLaunchKernelGGL(k_merge_partials<PP>, grid, block, 0, s, x->partial, S, rc, merged, tables); break;
    GS_MP_CASE(1) GS_MP_CASE(2) GS_MP_CASE(3) GS_MP_CASE(4) GS_MP_CASE(5) GS_MP_CASE(6) GS_MP_CASE(7) GS_MP_CASE(8)
    GS_MP_CASE(9) GS_MP_CASE(10) GS_MP_CASE(11) GS_MP_CASE(12) GS_MP_CASE(13) GS_MP_CASE(14) GS_MP_CASE(15)
    GS_MP_CASE(16)
#undef GS_MP_CASE
    default:
      hipLaunchKernelGGL(k_merge_partials_any, grid, block, 0, s, x->partial, S, rc, x->P, merged, tables);
      break;
  }
  return hipGetLastError();
}

}  // namespace gs
