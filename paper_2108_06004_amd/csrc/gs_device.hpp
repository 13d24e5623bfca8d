// gs_device.hpp -- device-side building blocks of the gs-SGD hot path (gfx950).
//
// Hashes: the Count Sketch bucket and sign families of the paper (Sec. III-A),
//   h_j(i) = ((a_j i + b_j) mod p) mod c,  s_j(i) = +1 iff ((a2_j i + b2_j) mod p) is odd,
// with p = 2^31 - 1. The mod-p step uses the Mersenne identity 2^31 = 1 (mod p), so a
// 62-bit product folds with shifts and adds; the mod-c step multiplies by a precomputed
// reciprocal (Granlund & Montgomery, "Division by invariant integers using
// multiplication", PLDI 1994, Thm 4.2): for 31-bit x and l = ceil(log2 c),
// m = ceil(2^(31+l) / c) < 2^32 gives floor(x / c) = floor(x m / 2^(31+l)).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace gs {

constexpr uint32_t kMersenne = 0x7fffffffu;
constexpr int kMaxRows = 16;
constexpr int kMaxWorkers = 64;

struct RowHash {
  uint32_t a, b;    // bucket hash
  uint32_t a2, b2;  // sign hash
};

// Kernel-argument copy of the hash family (uniform across the grid: scalar loads).
struct HashSet {
  RowHash row[kMaxRows];
  uint32_t c;      // columns
  uint32_t magic;  // ceil(2^(31+l) / c) with l = ceil(log2 c); 2^31 when c == 1 (l = 0)
  uint32_t shift;  // 31 + l
  int32_t r;       // rows
};

// The per-row constants a kernel keeps in registers for its hot loop.
struct RowConst {
  uint32_t a, b, a2, b2, c, magic, shift;
};

__device__ __forceinline__ RowConst row_const(const HashSet& hs, int j) {
  const RowHash rh = hs.row[j];
  return RowConst{rh.a, rh.b, rh.a2, rh.b2, hs.c, hs.magic, hs.shift};
}

// (a*i + b) mod p for a, b < p and i < 2^31.
__device__ __forceinline__ uint32_t mod_mersenne_affine(uint32_t a, uint32_t b, uint32_t i) {
  const uint64_t x = (uint64_t)a * i + b;                     // < 2^63
  const uint64_t y = (x & kMersenne) + (x >> 31);             // < 2^33
  const uint32_t z = (uint32_t)((y & kMersenne) + (y >> 31)); // <= 2^31 + 2
  return z >= kMersenne ? z - kMersenne : z;
}

// (x + y) mod p for x, y < p. Along a stride Δ of coordinates the affine hash advances by a
// constant, (a(i + Δ) + b) mod p = ((a i + b) mod p + (a Δ mod p)) mod p, so a loop over
// i, i + Δ, i + 2Δ, ... needs one multiply per row to start and one add per step after.
__device__ __forceinline__ uint32_t add_mod_mersenne(uint32_t x, uint32_t y) {
  const uint32_t s = x + y;  // < 2^32
  return s >= kMersenne ? s - kMersenne : s;
}

// x mod c for x < 2^31: q = floor(x * magic / 2^shift) is floor(x / c) exactly.
__device__ __forceinline__ uint32_t mod_c(uint32_t x, uint32_t c, uint32_t magic, uint32_t shift) {
  const uint32_t q = (uint32_t)(((uint64_t)x * magic) >> shift);
  return x - q * c;
}

// Column of coordinate i in a row, and the sign as a float sign-bit mask
// (0 for +1, 0x80000000 for -1).
__device__ __forceinline__ void hash_row(const RowConst& k, uint32_t i, uint32_t& col, uint32_t& sflip) {
  col = mod_c(mod_mersenne_affine(k.a, k.b, i), k.c, k.magic, k.shift);
  sflip = ((mod_mersenne_affine(k.a2, k.b2, i) & 1u) ^ 1u) << 31;
}

// Sign-bit mask of a raw sign-hash value: +1 (mask 0) iff the value is odd.
__device__ __forceinline__ uint32_t sign_flip_of(uint32_t raw2) { return ((raw2 & 1u) ^ 1u) << 31; }

__device__ __forceinline__ void hash_ij(const HashSet& hs, int j, uint32_t i, uint32_t& col, uint32_t& sflip) {
  hash_row(row_const(hs, j), i, col, sflip);
}

__device__ __forceinline__ float apply_sign(float x, uint32_t sflip) {
  return __uint_as_float(__float_as_uint(x) ^ sflip);
}

// Tree-order sum of P values held in x[0..P-1]: rounds of stride 1, 2, 4, ...; at stride s
// element m (a multiple of 2s) absorbs element m+s when it exists. This is the binomial
// tree of the paper's reduction: pairs (0,1),(2,3),... first, an unpaired highest rank
// passing through to the next round.
template <int P>
__device__ __forceinline__ float tree_sum(float (&x)[P]) {
#pragma unroll
  for (int s = 1; s < P; s <<= 1) {
#pragma unroll
    for (int m = 0; m + s < P; m += 2 * s) x[m] = x[m] + x[m + s];
  }
  return x[0];
}

// Runtime-P variant over a private array (used only when P is not one of the unrolled
// template instances).
__device__ __forceinline__ float tree_sum_dyn(float* x, int P) {
  for (int s = 1; s < P; s <<= 1)
    for (int m = 0; m + s < P; m += 2 * s) x[m] = x[m] + x[m + s];
  return x[0];
}

// Sorting network (odd-even transposition) over R registers, ascending.
template <int R>
__device__ __forceinline__ void sort_net(float (&v)[R]) {
#pragma unroll
  for (int pass = 0; pass < R; ++pass) {
#pragma unroll
    for (int t = pass & 1; t + 1 < R; t += 2) {
      const float lo = fminf(v[t], v[t + 1]);
      const float hi = fmaxf(v[t], v[t + 1]);
      v[t] = lo;
      v[t + 1] = hi;
    }
  }
}

template <int R>
__device__ __forceinline__ float median_sorted(const float (&v)[R]) {
  if constexpr (R & 1) {
    return v[R / 2];
  } else {
    const float s = v[R / 2 - 1] + v[R / 2];
    return s * 0.5f;
  }
}

// The estimate of coordinate i from a merged sketch (Alg. 2, query): the median over rows
// of s_j(i) * S[j][h_j(i)].
template <int R>
__device__ __forceinline__ float estimate_val(const RowConst (&kr)[R], const float* __restrict__ merged, uint32_t i) {
  float val[R];
#pragma unroll
  for (int j = 0; j < R; ++j) {
    uint32_t col, sflip;
    hash_row(kr[j], i, col, sflip);
    val[j] = apply_sign(merged[(int64_t)j * kr[j].c + col], sflip);
  }
  sort_net<R>(val);
  return median_sorted<R>(val);
}

// |x| as an order-preserving uint32 key (non-negative floats order like their bits).
__device__ __forceinline__ uint32_t abs_key(float x) { return __float_as_uint(x) & 0x7fffffffu; }

}  // namespace gs
