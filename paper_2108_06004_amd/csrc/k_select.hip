// k_select.hip -- HEAVYMIX estimate and selection (Alg. 2): the deterministic top-k and
// HEAVYMIX as printed.
//
// Estimate: est_i = median over rows of s_j(i) * S[j][h_j(i)] (register sorting network).
// Selection: the k largest keys, ties toward the lower index, output ascending. For the
// top-k the keys are the bit patterns of |est_i| (non-negative floats order like unsigned
// integers); for HEAVYMIX, heavy coordinates get 0x80000000 | bits(|est_i|) and the others
// their fill draw. The k-th key is found by a most-significant-digit radix select entirely
// on the device (no host synchronisation inside the call):
//   1. candidates: either every key reaching the pruned pass's sampled bound (k_sample ..
//      k_survivors: bound, heavy-cell bitmap, survivor estimates, with the candidates'
//      digit-1 histogram), or every coordinate, from the full estimate (k_unsketch /
//      k_unsketch_hm), which also runs whenever the pruned candidates fall short of k;
//   2. k_digit2 (many blocks): each block finds the digit-1 bucket (bits 31..20) of the
//      k-th key in the candidates' histogram; candidates in higher buckets are all taken and
//      set their bit in the output bitmap; digit 2 (bits 19..10) of the bucket's keys, and
//      the bucket compacted (keys and coordinates);
//   3. k_select2 (one block): digit 3 (bits 9..0) of the bucket gives the k-th key tau and
//      how many keys equal to tau are taken; if not all of them, the largest coordinate iota
//      taken among them (lowest coordinates win), by rank or by three index digits;
//   4. k_mark: the bucket's keys > tau, or == tau with index <= iota, set their bit;
//   5. k_emit: the bitmap is turned into ascending indices in one pass (each block counts
//      its words and takes its offset from the blocks before it by a decoupled look-back).
#include <algorithm>
#include <cmath>
#include <type_traits>

#include "gs_internal.hpp"

namespace gs {
namespace {

constexpr int kBlock = 256;
constexpr int kSelBlock = 1024;
constexpr int kEmitWordsPerThread = 4;
constexpr int kEmitWordsPerBlock = kSelBlock * kEmitWordsPerThread;

int grid_for(int64_t work_items, int per_block, int cap) {
  int64_t b = (work_items + per_block - 1) / per_block;
  if (b < 1) b = 1;
  if (b > cap) b = cap;
  return (int)b;
}

// Inclusive prefix sum of x over the threads of a block of BS threads (BS a multiple of 64,
// at most 64 waves). sh must hold BS/64 words. All threads must call it.
template <int BS>
__device__ uint32_t block_scan_incl(uint32_t x, uint32_t* sh, uint32_t& total) {
  constexpr int kWaves = BS / 64;
  const int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) {
    const uint32_t y = __shfl_up(x, o, 64);
    if (lane >= o) x += y;
  }
  if (lane == 63) sh[wid] = x;
  __syncthreads();
  if (wid == 0) {
    uint32_t w = lane < kWaves ? sh[lane] : 0u;
#pragma unroll
    for (int o = 1; o < 64; o <<= 1) {
      const uint32_t y = __shfl_up(w, o, 64);
      if (lane >= o) w += y;
    }
    if (lane < kWaves) sh[lane] = w;
  }
  __syncthreads();
  total = sh[kWaves - 1];
  const uint32_t add = wid ? sh[wid - 1] : 0u;
  __syncthreads();
  return x + add;
}

// Scan the histogram h[NB] (LDS or global; NB a multiple of BS, at most 16 bins per
// thread) in descending or ascending bin order and find the first bin at which the running
// count reaches `need` (1 <= need <= total). res[0] = that bin, res[1] = count in the bins
// before it (in scan order). Each thread reads its bins once. All threads must call it.
template <int BS, int NB>
__device__ void find_bucket(const uint32_t* h, bool descending, uint32_t need, uint32_t* shw, uint32_t* res) {
  constexpr int kPer = NB / BS;
  static_assert(kPer >= 1 && kPer * BS == NB && kPer <= 16, "bins per thread");
  uint32_t cnt[kPer];
  uint32_t sum = 0;
#pragma unroll
  for (int m = 0; m < kPer; ++m) {
    const int pos = threadIdx.x * kPer + m;
    cnt[m] = h[descending ? NB - 1 - pos : pos];
    sum += cnt[m];
  }
  uint32_t total;
  const uint32_t incl = block_scan_incl<BS>(sum, shw, total);
  const uint32_t excl = incl - sum;
  if (excl < need && need <= incl) {
    uint32_t run = excl;
    for (int m = 0; m < kPer; ++m) {
      if (run + cnt[m] >= need) {
        const int pos = threadIdx.x * kPer + m;
        res[0] = (uint32_t)(descending ? NB - 1 - pos : pos);
        res[1] = run;
        break;
      }
      run += cnt[m];
    }
  }
  __syncthreads();
}

// Adds 1 to the LDS histogram bin `bin` of every lane with `take` set; every lane of the
// wave must call it. The lanes whose bin equals that of the first taking lane add with one
// atomic, so runs of equal keys (all-zero estimates, say) do not serialise on one address.
__device__ __forceinline__ void hist_add(uint32_t* h, bool take, uint32_t bin) {
  const uint64_t act = __ballot(take);
  if (act == 0ull) return;
  const int first = __builtin_ctzll(act);
  const uint32_t b0 = __shfl(bin, first, 64);
  const uint64_t same = __ballot(take && bin == b0);
  if (take && bin != b0) atomicAdd(&h[bin], 1u);
  if ((int)(threadIdx.x & 63) == first) atomicAdd(&h[b0], (uint32_t)__popcll(same));
}

// ------------------------------------------------------------------------------------
// Step 1, full path: every coordinate is a candidate ("dense" candidates: candidate t is
// coordinate t, so no index array). The estimate, its key in cand_key[i], the digit-1
// histogram in hist, and the output bitmap cleared.

// After a pruned pass: true when fewer than k coordinates reached its bound, so the full
// estimate has to run. The first kernel of the full path calls it (every block sees the
// same counts) and raises ctl->fallback, which gates the kernels after it.
__device__ __forceinline__ bool fallback_needed(SelectCtl* ctl) {
  const bool fb = ctl->n_cand < ctl->k;
  if (fb && blockIdx.x == 0 && threadIdx.x == 0) ctl->fallback = 1u;
  return fb;
}

// k_unsketch's grid. Each block adds its LDS histogram into the global one with an atomic
// per non-empty bin, and the atomics of many blocks on the few well-filled bins queue at one
// address each. Up to kUnsketchSmall * kBlock * (CUs) coordinates that queue costs more than
// the blocks' parallelism gains: at most one block per CU then, each thread taking two
// coordinates per pass with all their cell loads in flight. Beyond it, four blocks per CU,
// one coordinate per thread per pass.
constexpr int kUnsketchSmall = 8;

template <int R, int U>
__global__ void __launch_bounds__(kBlock) k_unsketch(HashSet hs, const float* __restrict__ merged, int64_t d,
                                                     float* __restrict__ est, uint32_t* __restrict__ keys,
                                                     uint32_t* __restrict__ hist, uint32_t* __restrict__ bitmap,
                                                     SelectCtl* __restrict__ gate) {
  if (gate && !fallback_needed(gate)) return;  // the pruned selection sufficed
  __shared__ uint32_t h[kDigit1Bins];
  for (int b = threadIdx.x; b < kDigit1Bins; b += kBlock) h[b] = 0u;
  RowConst kr[R];
#pragma unroll
  for (int j = 0; j < R; ++j) kr[j] = row_const(hs, j);
  __syncthreads();
  const int64_t stride = (int64_t)gridDim.x * kBlock;
  const int64_t i0 = (int64_t)blockIdx.x * kBlock + threadIdx.x;
  uint32_t hb[R], hsg[R], db[R], dsg[R];  // raw hashes of the current i and their per-stride steps
#pragma unroll
  for (int j = 0; j < R; ++j) {
    hb[j] = mod_mersenne_affine(kr[j].a, kr[j].b, (uint32_t)i0);
    hsg[j] = mod_mersenne_affine(kr[j].a2, kr[j].b2, (uint32_t)i0);
    db[j] = mod_mersenne_affine(kr[j].a, 0u, (uint32_t)stride);
    dsg[j] = mod_mersenne_affine(kr[j].a2, 0u, (uint32_t)stride);
  }
  // U coordinates (i, i + stride, ...) per pass with all their cell loads in flight; a cell
  // column is valid for any hash value, so the loads past d need no guard
  for (int64_t ib = i0; ib < d; ib += U * stride) {
    float val[U][R];
#pragma unroll
    for (int u = 0; u < U; ++u) {
#pragma unroll
      for (int j = 0; j < R; ++j) {
        const uint32_t col = mod_c(hb[j], kr[j].c, kr[j].magic, kr[j].shift);
        val[u][j] = apply_sign(merged[(int64_t)j * hs.c + col], sign_flip_of(hsg[j]));
        hb[j] = add_mod_mersenne(hb[j], db[j]);
        hsg[j] = add_mod_mersenne(hsg[j], dsg[j]);
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int64_t i = ib + u * stride;
      if (i >= d) break;
      sort_net<R>(val[u]);
      const float e = median_sorted<R>(val[u]);
      if (est) est[i] = e;
      const uint32_t key = abs_key(e);
      keys[i] = key;
      atomicAdd(&h[key >> kDigit1Shift], 1u);
      if ((i & 31) == 0) bitmap[i >> 5] = 0u;
    }
  }
  __syncthreads();
  for (int b = threadIdx.x; b < kDigit1Bins; b += kBlock) {
    const uint32_t n = h[b];
    if (n) atomicAdd(&hist[b], n);
  }
}

// ------------------------------------------------------------------------------------
// Steps 2 and 3: digits 2 and 3 of the k-th key, then the index cut among equal keys.
// Candidates are either the pruned pass's (keys in cand_key, coordinates in cand_idx,
// digit-1 histogram in hist_c) or dense (after the full estimate: every coordinate, key
// in cand_key, histogram in hist). dense_cands() tells which.

constexpr int kSelUnroll = 8;    // candidate loads in flight per thread
constexpr int kTieMax = 1024;    // ties at the k-th key resolved by ranking in LDS (else radix digits)
constexpr int kDigit2Block = 1024;              // threads per k_digit2 block
constexpr int kStageBuf = 8 * kDigit2Block;  // per-block LDS buffer of k_digit2 (keys and coordinates)

__device__ __forceinline__ bool dense_cands(const SelectCtl* ctl, int pruned) {
  return !pruned || ctl->fallback != 0u;
}

// Step 2 (many blocks): every block finds the digit-1 bucket b1 of the k-th key in the
// candidates' histogram (block 0 records it); then the digit-2 histogram of the bucket's
// keys (LDS per block, added into hist2) and the bucket compacted, key and coordinate, into
// stage_key / stage_idx (an LDS buffer per block, one global atomic per flush).
__global__ void __launch_bounds__(kDigit2Block) k_digit2(const uint32_t* __restrict__ cand_key,
                                                   const int32_t* __restrict__ cand_idx,
                                                   SelectCtl* __restrict__ ctl, int64_t cap, int64_t d,
                                                   const uint32_t* __restrict__ hist_c,
                                                   const uint32_t* __restrict__ hist, int pruned, uint32_t k,
                                                   uint32_t* __restrict__ hist2, uint32_t* __restrict__ stage_key,
                                                   int32_t* __restrict__ stage_idx, uint32_t* __restrict__ bitmap) {
  __shared__ uint32_t h[kDigitBins];
  __shared__ uint32_t bkey[kStageBuf];
  __shared__ int32_t bidx[kStageBuf];
  __shared__ uint32_t shw[kDigit2Block / 64];
  __shared__ uint32_t res[2];
  __shared__ uint32_t bn, gbase;
  const bool dense = dense_cands(ctl, pruned);
  const int64_t n = dense ? d : (ctl->n_cand < (uint64_t)cap ? (int64_t)ctl->n_cand : cap);
  find_bucket<kDigit2Block, kDigit1Bins>(dense ? hist : hist_c, true, k, shw, res);
  const uint32_t b1 = res[0];
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    ctl->b1 = res[0];
    ctl->above1 = res[1];
  }
  const int lane = threadIdx.x & 63;
  for (int b = threadIdx.x; b < kDigitBins; b += kDigit2Block) h[b] = 0u;
  if (threadIdx.x == 0) bn = 0u;
  __syncthreads();
  const int64_t per = (n + gridDim.x - 1) / gridDim.x;
  const int64_t lo = (int64_t)blockIdx.x * per, hi = min(n, lo + per);
  constexpr int V = 4;
  for (int64_t c0 = lo; c0 < hi; c0 += (int64_t)V * kDigit2Block) {  // block-uniform
    uint32_t key[V];
#pragma unroll
    for (int m = 0; m < V; ++m) {
      const int64_t t = c0 + (int64_t)m * kDigit2Block + threadIdx.x;
      key[m] = t < hi ? cand_key[t] : 0u;
    }
#pragma unroll
    for (int m = 0; m < V; ++m) {
      const int64_t t = c0 + (int64_t)m * kDigit2Block + threadIdx.x;
      const uint32_t d1 = key[m] >> kDigit1Shift;
      if (t < hi && d1 > b1) {  // above the k-th key's bucket: taken
        const uint32_t ix = dense ? (uint32_t)t : (uint32_t)cand_idx[t];
        atomicOr(&bitmap[ix >> 5], 1u << (ix & 31u));
      }
      const bool take = t < hi && d1 == b1;
      hist_add(h, take, (key[m] >> 10) & 1023u);
      const uint64_t bal = __ballot(take);
      uint32_t wbase = 0u;
      if (lane == 0 && bal) wbase = atomicAdd(&bn, (uint32_t)__popcll(bal));
      wbase = __shfl(wbase, 0);
      if (take) {
        const uint32_t pos = wbase + (uint32_t)__popcll(bal & ((1ull << lane) - 1ull));
        bkey[pos] = key[m];
        bidx[pos] = dense ? (int32_t)t : cand_idx[t];
      }
    }
    __syncthreads();
    const uint32_t nb = bn;  // < kStageBuf / 2 + V * kDigit2Block <= kStageBuf
    if (nb >= (uint32_t)(kStageBuf / 2) || (c0 + (int64_t)V * kDigit2Block >= hi && nb > 0)) {
      if (threadIdx.x == 0) gbase = atomicAdd(&ctl->n_stage2, nb);
      __syncthreads();
      const uint32_t g0 = gbase;
      for (uint32_t t = threadIdx.x; t < nb; t += kDigit2Block) {
        stage_key[g0 + t] = bkey[t];
        stage_idx[g0 + t] = bidx[t];
      }
      __syncthreads();
      if (threadIdx.x == 0) bn = 0u;
    }
    __syncthreads();
  }
  for (int b = threadIdx.x; b < kDigitBins; b += kDigit2Block) {
    const uint32_t c = h[b];
    if (c) atomicAdd(&hist2[b], c);
  }
}

// Step 3 (one block): the digit-2 bucket from the histogram, digit 3 over the staged keys,
// and the index cut among the staged keys equal to tau. Clears the histograms it and
// k_digit2 consumed for the next call.
__global__ void __launch_bounds__(kSelBlock) k_select2(SelectCtl* __restrict__ ctl, uint32_t* __restrict__ hist2,
                                                       const uint32_t* __restrict__ stage_key,
                                                       const int32_t* __restrict__ stage_idx,
                                                       uint32_t* __restrict__ hist_c, uint32_t* __restrict__ hist,
                                                       int pruned, uint32_t k, unsigned long long* __restrict__ flags,
                                                       int64_t emit_blocks) {
  __shared__ uint32_t h[2048];
  __shared__ uint32_t shw[kSelBlock / 64];
  __shared__ uint32_t res[2];
  __shared__ uint32_t n_tie;
  const int64_t n2 = ctl->n_stage2;
  const uint32_t b1 = ctl->b1;
  const uint32_t need1 = k - ctl->above1;
  const bool dense = dense_cands(ctl, pruned);

  // digit 2 (key bits 19..10) among keys in bucket b1, scanned from the top
  for (int b = threadIdx.x; b < kDigitBins; b += kSelBlock) {
    h[b] = hist2[b];
    hist2[b] = 0u;
  }
  if (pruned)
    for (int b = threadIdx.x; b < kDigit1Bins; b += kSelBlock) hist_c[b] = 0u;
  if (dense)
    for (int b = threadIdx.x; b < kDigit1Bins; b += kSelBlock) hist[b] = 0u;
  for (int64_t b = threadIdx.x; b < emit_blocks; b += kSelBlock) flags[b] = 0ull;  // the emit's look-back words
  __syncthreads();
  find_bucket<kSelBlock, kDigitBins>(h, true, need1, shw, res);
  const uint32_t pre2 = (b1 << 10) | res[0];
  const uint32_t need2 = need1 - res[1];
  __syncthreads();

  // digit 3 (key bits 9..0) among the staged keys with the 22-bit prefix pre2
  for (int b = threadIdx.x; b < kDigitBins; b += kSelBlock) h[b] = 0u;
  __syncthreads();
  for (int64_t t0 = 0; t0 < n2; t0 += (int64_t)kSelUnroll * kSelBlock) {
    uint32_t key[kSelUnroll];
#pragma unroll
    for (int m = 0; m < kSelUnroll; ++m) {
      const int64_t t = t0 + (int64_t)m * kSelBlock + threadIdx.x;
      key[m] = t < n2 ? stage_key[t] : 0u;
    }
#pragma unroll
    for (int m = 0; m < kSelUnroll; ++m) {
      const int64_t t = t0 + (int64_t)m * kSelBlock + threadIdx.x;
      hist_add(h, t < n2 && (key[m] >> 10) == pre2, key[m] & 1023u);
    }
  }
  __syncthreads();
  find_bucket<kSelBlock, kDigitBins>(h, true, need2, shw, res);
  const uint32_t tau = (pre2 << 10) | res[0];
  const uint32_t need3 = need2 - res[1];  // how many keys equal to tau are taken
  const uint32_t n_eq = h[res[0]];
  __syncthreads();

  // every key equal to tau is in the stage (its digit 1 is b1)
  uint32_t iota = 0x7fffffffu;
  if (need3 < n_eq && n_eq <= kTieMax) {
    // few keys equal to tau (the usual case: an estimate is one table cell): one pass
    // collects their coordinates in LDS, and iota is the one with exactly need3 - 1 smaller
    // (the coordinates are distinct)
    if (threadIdx.x == 0) n_tie = 0u;
    __syncthreads();
    for (int64_t t0 = 0; t0 < n2; t0 += (int64_t)kSelUnroll * kSelBlock) {
      uint32_t key[kSelUnroll];
#pragma unroll
      for (int m = 0; m < kSelUnroll; ++m) {
        const int64_t t = t0 + (int64_t)m * kSelBlock + threadIdx.x;
        key[m] = t < n2 ? stage_key[t] : 0u;
      }
#pragma unroll
      for (int m = 0; m < kSelUnroll; ++m) {
        const int64_t t = t0 + (int64_t)m * kSelBlock + threadIdx.x;
        if (t < n2 && key[m] == tau) {
          const uint32_t pos = atomicAdd(&n_tie, 1u);
          if (pos < (uint32_t)kTieMax) h[pos] = (uint32_t)stage_idx[t];
        }
      }
    }
    __syncthreads();
    const uint32_t m_tie = min(n_tie, (uint32_t)kTieMax);  // == n_eq
    for (uint32_t a = threadIdx.x; a < m_tie; a += kSelBlock) {
      const uint32_t xa = h[a];
      uint32_t rank = 0;
      for (uint32_t b = 0; b < m_tie; ++b) rank += h[b] < xa ? 1u : 0u;
      if (rank == need3 - 1) res[0] = xa;
    }
    __syncthreads();
    iota = res[0];
  } else if (need3 < n_eq) {
    // many ties: ascending index digits among keys equal to tau: bits 30..21, 20..10, 9..0
    for (int b = threadIdx.x; b < 1024; b += kSelBlock) h[b] = 0u;
    __syncthreads();
    for (int64_t t0 = 0; t0 < n2; t0 += kSelBlock) {  // block-uniform
      const int64_t t = t0 + threadIdx.x;
      const bool tie = t < n2 && stage_key[t] == tau;
      hist_add(h, tie, tie ? (uint32_t)stage_idx[t] >> 21 : 0u);
    }
    __syncthreads();
    find_bucket<kSelBlock, 1024>(h, false, need3, shw, res);
    const uint32_t c1 = res[0];
    const uint32_t needc = need3 - res[1];
    __syncthreads();

    for (int b = threadIdx.x; b < 2048; b += kSelBlock) h[b] = 0u;
    __syncthreads();
    for (int64_t t0 = 0; t0 < n2; t0 += kSelBlock) {
      const int64_t t = t0 + threadIdx.x;
      const uint32_t ix = t < n2 && stage_key[t] == tau ? (uint32_t)stage_idx[t] : 0xffffffffu;
      const bool in = ix != 0xffffffffu && (ix >> 21) == c1;
      hist_add(h, in, (ix >> 10) & 2047u);
    }
    __syncthreads();
    find_bucket<kSelBlock, 2048>(h, false, needc, shw, res);
    const uint32_t pre_i = (c1 << 11) | res[0];
    const uint32_t needd = needc - res[1];
    __syncthreads();

    for (int b = threadIdx.x; b < 1024; b += kSelBlock) h[b] = 0u;
    __syncthreads();
    for (int64_t t0 = 0; t0 < n2; t0 += kSelBlock) {
      const int64_t t = t0 + threadIdx.x;
      const uint32_t ix = t < n2 && stage_key[t] == tau ? (uint32_t)stage_idx[t] : 0xffffffffu;
      const bool in = ix != 0xffffffffu && (ix >> 10) == pre_i;
      hist_add(h, in, ix & 1023u);
    }
    __syncthreads();
    find_bucket<kSelBlock, 1024>(h, false, needd, shw, res);
    iota = (pre_i << 10) | res[0];
  }
  if (threadIdx.x == 0) {
    ctl->tau = tau;
    ctl->iota = iota;
    ctl->n_staged = (uint32_t)n2;
    ctl->n_stage2 = 0u;
    ctl->emit_ticket = 0u;
  }
}

// ------------------------------------------------------------------------------------
// Step 4: mark the taken keys of the staged digit-1 bucket (the candidates above it set
// their bits in k_digit2).

__global__ void __launch_bounds__(kBlock) k_mark(const uint32_t* __restrict__ stage_key,
                                                 const int32_t* __restrict__ stage_idx,
                                                 const SelectCtl* __restrict__ ctl, uint32_t* __restrict__ bitmap) {
  const int64_t n2 = ctl->n_staged;
  const uint32_t tau = ctl->tau, iota = ctl->iota;
  const int64_t stride = (int64_t)gridDim.x * kBlock;
  for (int64_t t = (int64_t)blockIdx.x * kBlock + threadIdx.x; t < n2; t += stride) {
    const uint32_t key = stage_key[t];
    if (key < tau) continue;
    const uint32_t ix = (uint32_t)stage_idx[t];
    if (key > tau || ix <= iota) atomicOr(&bitmap[ix >> 5], 1u << (ix & 31u));
  }
}

// ------------------------------------------------------------------------------------
// Pruned estimate (used when no estimate vector is requested). A coordinate whose median
// over rows has |est| >= tau0 has at least ceil(r/2) cells with |cell| >= tau0 (odd r: the
// median and the values beyond it; even r: the upper (or lower) half, since
// fl(fl(m1 + m2) * 0.5) never exceeds m2 in magnitude). So with tau0 no larger than the
// k-th |est|, only coordinates with ceil(r/2) "heavy" cells can be selected, and a bitmap
// of heavy cells replaces most table reads. tau0 is the rho-th largest of M sampled exact
// estimates, rho ~ 2 M k / d plus a margin; if fewer than k coordinates reach tau0 the
// unpruned kernels (gated on ctl->fallback) redo the selection, so the result is exact
// either way.

template <int R>
__device__ __forceinline__ uint32_t estimate_key(const RowConst (&kr)[R], const float* __restrict__ merged,
                                                 uint32_t i) {
  return abs_key(estimate_val<R>(kr, merged, i));
}

// Sampled keys at M evenly spaced coordinates: |est| keys, or (HEAVYMIX) the fill keys
// rnd >> 1, whose rho-th largest bounds the fill from below. Their digit-1 histogram is
// added into hist_s for k_heavy's bound.
template <int R, bool HM>
__global__ void __launch_bounds__(kBlock) k_sample(HashSet hs, const float* __restrict__ merged, int64_t d, int M,
                                                   const uint32_t* __restrict__ rnd, uint32_t* __restrict__ out,
                                                   uint32_t* __restrict__ hist_s) {
  __shared__ uint32_t h[kDigit1Bins];
  for (int b = threadIdx.x; b < kDigit1Bins; b += kBlock) h[b] = 0u;
  __syncthreads();
  const int s = blockIdx.x * kBlock + threadIdx.x;
  const bool ok = s < M;
  uint32_t key = 0u;
  if (ok) {
    const uint32_t i = (uint32_t)(((int64_t)s * d) / M);
    if constexpr (HM) {
      key = rnd[i] >> 1;
    } else {
      RowConst kr[R];
#pragma unroll
      for (int j = 0; j < R; ++j) kr[j] = row_const(hs, j);
      key = estimate_key<R>(kr, merged, i);
    }
    out[s] = key;
  }
  hist_add(h, ok, key >> kDigit1Shift);
  __syncthreads();
  for (int b = threadIdx.x; b < kDigit1Bins; b += kBlock) {
    const uint32_t c = h[b];
    if (c) atomicAdd(&hist_s[b], c);
  }
}

// tau0 = the rho-th largest sampled key, found by one block of BS threads: digit 1 from
// k_sample's histogram hist_s, digits 2 and 3 over the sampled keys held in registers. h is
// an LDS histogram of kDigitBins words. All threads must call it; each gets tau0.
template <int BS>
__device__ uint32_t sampled_bound(const uint32_t* __restrict__ sample, int M, uint32_t rho,
                                  const uint32_t* __restrict__ hist_s, uint32_t* h, uint32_t* shw, uint32_t* res) {
  constexpr int kPer = kSampleMax / BS;
  uint32_t key[kPer];
#pragma unroll
  for (int m = 0; m < kPer; ++m) {
    const int t = m * BS + threadIdx.x;
    key[m] = t < M ? sample[t] : 0u;
  }
  for (int b = threadIdx.x; b < kDigitBins; b += BS) h[b] = 0u;
  find_bucket<BS, kDigit1Bins>(hist_s, true, rho, shw, res);
  const uint32_t b1 = res[0], need2 = rho - res[1];
#pragma unroll
  for (int m = 0; m < kPer; ++m) {
    const bool take = m * BS + (int)threadIdx.x < M && (key[m] >> kDigit1Shift) == b1;
    hist_add(h, take, (key[m] >> 10) & 1023u);
  }
  __syncthreads();
  find_bucket<BS, kDigitBins>(h, true, need2, shw, res);
  const uint32_t pre = (b1 << 10) | res[0], need3 = need2 - res[1];
  for (int b = threadIdx.x; b < kDigitBins; b += BS) h[b] = 0u;
  __syncthreads();
#pragma unroll
  for (int m = 0; m < kPer; ++m) {
    const bool take = m * BS + (int)threadIdx.x < M && (key[m] >> 10) == pre;
    hist_add(h, take, key[m] & 1023u);
  }
  __syncthreads();
  find_bucket<BS, kDigitBins>(h, true, need3, shw, res);
  return (pre << 10) | res[0];
}

// Heavy-cell bitmap: bit j * hrow + col (rows padded to hrow bits, a multiple of 64, so a
// row starts on a word) is |merged[j][col]| >= tau0, or (HEAVYMIX,
// hm = 1) merged[j][col]^2 >= theta in fp64 (one ballot per 64 cells); with hm the sampled fill
// bound tau0 is still found here, for the pruned pass. A coordinate with
// est^2 >= theta has ceil(r/2) cells with |cell| >= |est| (see the pruned pass), and the
// squares of fp32 values are exact in fp64, so those cells pass the same test.
// Every block first finds tau0 itself (the sampled keys are read from L2; block 0 records
// it and resets the selection counters), so no single-block kernel runs in between.
constexpr int kHeavyUnroll = 8;  // 64-cell groups per wave and pass of k_heavy
__global__ void __launch_bounds__(kSelBlock) k_heavy(const float* __restrict__ merged, int64_t c, int64_t hrow,
                                                  int r,
                                                  SelectCtl* __restrict__ ctl, uint32_t* __restrict__ heavy,
                                                  int hm, const uint32_t* __restrict__ sample, int M,
                                                  uint32_t rho, uint32_t k, const uint32_t* __restrict__ hist_s) {
  __shared__ uint32_t h[kDigitBins];
  __shared__ uint32_t shw[kSelBlock / 64];
  __shared__ uint32_t res[2];
  const uint32_t tau0 = sampled_bound<kSelBlock>(sample, M, rho, hist_s, h, shw, res);
  if (blockIdx.x == 0 && threadIdx.x == 0) {
    ctl->tau0 = tau0;
    ctl->k = k;
    ctl->n_cand = 0u;
    ctl->n_surv = 0u;
    ctl->fallback = 0u;
  }
  const double theta = ctl->theta;
  // The map in groups of 64 cells (one ballot, two words each; hrow is a multiple of 64, so a
  // group lies in one row). A wave takes UH consecutive groups per pass with all their loads
  // in flight together. r <= 16 and hrow <= 2^31 keep group indices below 2^29.
  constexpr int UH = kHeavyUnroll;
  const uint32_t gpr = (uint32_t)(hrow >> 6);  // groups per row
  const int64_t ng = ((int64_t)r * hrow) >> 6;
  const int lane = threadIdx.x & 63;
  // wave index, the same in every lane (a scalar)
  const int64_t wv = __builtin_amdgcn_readfirstlane((uint32_t)(((int64_t)blockIdx.x * kSelBlock + threadIdx.x) >> 6));
  const int64_t nwv = ((int64_t)gridDim.x * kSelBlock) >> 6;
  for (int64_t g0 = wv * UH; g0 < ng; g0 += nwv * UH) {
    float x[UH];
    bool in[UH];
    // row j and group-in-row rr of group g0 + q, advanced one group at a time
    uint32_t j = (uint32_t)g0 / gpr, rr = (uint32_t)g0 - j * gpr;
#pragma unroll
    for (int q = 0; q < UH; ++q) {
      const int64_t col = (int64_t)rr * 64 + lane;
      in[q] = g0 + q < ng && col < c;
      x[q] = in[q] ? merged[(int64_t)j * c + col] : 0.f;
      if (++rr == gpr) {
        rr = 0;
        ++j;
      }
    }
#pragma unroll
    for (int q = 0; q < UH; ++q) {
      const bool hv = in[q] && (hm ? (double)x[q] * (double)x[q] >= theta : abs_key(x[q]) >= tau0);
      const uint64_t m = __ballot(hv);
      if (lane == 0 && g0 + q < ng) {
        heavy[2 * (g0 + q)] = (uint32_t)m;
        heavy[2 * (g0 + q) + 1] = (uint32_t)(m >> 32);
      }
    }
  }
}

// Coarse heavy-cell map: coarse word w covers fine words [w*G, w*G + G) (G = 2^log2g <= 32);
// each fine word contributes 32/G bits, bit q set when any of its cells q*G .. q*G+G-1 is.
__global__ void __launch_bounds__(kBlock) k_coarse(const uint32_t* __restrict__ fine, int64_t fine_words,
                                                   int log2g, uint32_t* __restrict__ coarse, int64_t coarse_words) {
  const int G = 1 << log2g;
  const int per = 32 / G;  // coarse bits from one fine word
  const uint32_t mask = G == 32 ? 0xffffffffu : ((1u << G) - 1u);
  const int64_t stride = (int64_t)gridDim.x * kBlock;
  for (int64_t w = (int64_t)blockIdx.x * kBlock + threadIdx.x; w < coarse_words; w += stride) {
    uint32_t out = 0u;
    for (int f = 0; f < G; ++f) {
      const int64_t fw = w * G + f;
      const uint32_t x = fw < fine_words ? fine[fw] : 0u;
      for (int q = 0; q < per; ++q)
        if ((x >> (q * G)) & mask) out |= 1u << (f * per + q);
    }
    coarse[w] = out;
  }
}

// The pruned pass, in two kernels.
// k_pruned: every coordinate checks its r heavy bits (bitmap in LDS when it fits); the
// survivors (ceil(r/2) heavy cells; for HEAVYMIX also every coordinate whose fill key
// rnd[i] >> 1 reaches tau0) are queued -- through an LDS buffer, one global atomic per
// flush -- and the output bitmap words are cleared on the way.
// k_survivors: the queued coordinates, with every lane busy, compute their exact estimate
// and append the candidates (key >= tau0; for HEAVYMIX heavy ones always, key
// 0x80000000 | bits(|est|), others by their fill key) and count |H|. Splitting keeps the
// table reads of the few survivors from stalling whole waves of the first pass.
// dynamic LDS of k_pruned: [map words?][buf indices]
constexpr int kPruneBlock = 1024;  // 16 waves per CU; the heavy bitmap fills the LDS

// Where the pruned pass finds a cell's heavy bit. The map's address space is fixed at
// compile time so that LDS lookups are LDS instructions, not generic ones.
constexpr int kMapFine = 0;    // the fine map (one bit per cell), copied into LDS
constexpr int kMapCoarse = 1;  // a coarse map in LDS (one bit per 2^coarse_log2 cells, set when
                               // any of them is heavy); a set bit is confirmed in the fine map
                               // in global memory, so the count equals the fine map's
constexpr int kMapGlobal = 2;  // the fine map read from global memory

constexpr int kPruneLdsWords = 160 * 1024 / 4;  // the whole LDS of a CU (one workgroup per CU)

template <int MAP>
__device__ __forceinline__ int64_t map_words_in_lds(int64_t map_words) {
  return MAP == kMapGlobal ? 0 : map_words;
}

// Bit e & 31 of word w (the hardware takes the low five bits of the offset).
__device__ __forceinline__ uint32_t bit_at(uint32_t w, uint32_t e) { return __builtin_amdgcn_ubfe(w, e, 1u); }

template <int R, bool HM, int MAP>
__global__ void __launch_bounds__(kPruneBlock) k_pruned(HashSet hs, int64_t d, SelectCtl* __restrict__ ctl,
                                                   const uint32_t* __restrict__ heavy,
                                                   const uint32_t* __restrict__ lmap, int64_t map_words,
                                                   int64_t hrow, int coarse_log2, int buf_cap,
                                                   uint32_t* __restrict__ queue,
                                                   uint32_t* __restrict__ bitmap, const uint32_t* __restrict__ rnd,
                                                   uint32_t* __restrict__ hist_s) {
  // coordinates per lane per pass: independent hash chains in flight (two registers each per
  // row, so fewer with many rows, where four would spill); six with the map in LDS and few
  // rows (d = 25.6M x 8, r = 5: 71 -> 68.5 us; with the coarse map six measured no better)
  constexpr int U = (MAP == kMapFine && R <= 6) ? 6 : R <= 8 ? 4 : R <= 12 ? 2 : 1;
  // map index j * hrow + col of a cell; below 2^32 whenever a map fits in LDS
  using Cell = typename std::conditional<MAP == kMapGlobal, uint64_t, uint32_t>::type;
  // LDS: [map words][buf_cap queue entries][2 counters], one static array, so a lookup's
  // address is known at compile time to need no base added
  __shared__ uint32_t sm[kPruneLdsWords];
  uint32_t& bn = sm[map_words_in_lds<MAP>(map_words) + buf_cap];
  uint32_t& gbase = sm[map_words_in_lds<MAP>(map_words) + buf_cap + 1];
  if (blockIdx.x == 0)  // the samples' histogram, read by k_heavy, cleared for the next call
    for (int b = threadIdx.x; b < kDigit1Bins; b += kPruneBlock) hist_s[b] = 0u;
  uint32_t* buf = sm;
  if constexpr (MAP != kMapGlobal) {
    // map_words is even and the map 8-byte aligned: copy 16 bytes per lane, 8 loads in flight
    const int64_t n4 = map_words / 4;
    const uint4* src = reinterpret_cast<const uint4*>(lmap);
    uint4* dst = reinterpret_cast<uint4*>(sm);
    int64_t w = threadIdx.x;
    for (; w + 7 * kPruneBlock < n4; w += 8 * kPruneBlock) {
      uint4 t[8];
#pragma unroll
      for (int m = 0; m < 8; ++m) t[m] = src[w + m * kPruneBlock];
#pragma unroll
      for (int m = 0; m < 8; ++m) dst[w + m * kPruneBlock] = t[m];
    }
    for (; w < n4; w += kPruneBlock) dst[w] = src[w];
    for (int64_t x = 4 * n4 + threadIdx.x; x < map_words; x += kPruneBlock) sm[x] = lmap[x];
    buf = sm + map_words;
  }
  RowConst kr[R];
#pragma unroll
  for (int j = 0; j < R; ++j) kr[j] = row_const(hs, j);
  const uint32_t tau0 = ctl->tau0;
  constexpr int need = (R + 1) / 2;
  if (threadIdx.x == 0) bn = 0;
  __syncthreads();
  const int64_t stride = (int64_t)gridDim.x * kPruneBlock * U;
  const int64_t base0 = (int64_t)blockIdx.x * kPruneBlock * U;
  // Raw bucket hashes and columns of this lane's U coordinates, advanced by one stride per
  // pass without a multiply: the raw hash moves by db = (a * stride) mod p, less p when it
  // passes p, so the column moves by dc1 = db mod c, or by dc2 = (db - p) mod c after such a
  // wrap, and is brought back below c by one subtraction. The raw hash is kept biased by
  // kBias = 2^32 - p, so that passing p is the carry out of the 32-bit add.
  constexpr uint32_t kBias = 0x80000001u;
  uint32_t hb[R][U], cb[R][U], db[R], dc1[R], dc2[R];
  const uint32_t pc = mod_c(kMersenne, kr[0].c, kr[0].magic, kr[0].shift);  // p mod c
#pragma unroll
  for (int j = 0; j < R; ++j) {
    db[j] = mod_mersenne_affine(kr[j].a, 0u, (uint32_t)stride);
    dc1[j] = mod_c(db[j], kr[j].c, kr[j].magic, kr[j].shift);
    dc2[j] = dc1[j] >= pc ? dc1[j] - pc : dc1[j] + (kr[j].c - pc);
    // the select between the two steps takes one operand from a vector register: keep both
    // there for the whole kernel rather than copying them in every pass
    asm volatile("" : "+v"(dc1[j]), "+v"(dc2[j]));
#pragma unroll
    for (int m = 0; m < U; ++m) {
      const uint32_t raw =
          mod_mersenne_affine(kr[j].a, kr[j].b, (uint32_t)(base0 + threadIdx.x + (int64_t)m * kPruneBlock));
      hb[j][m] = raw + kBias;  // < 2^32: raw < p
      cb[j][m] = mod_c(raw, kr[j].c, kr[j].magic, kr[j].shift);
    }
  }
  auto advance = [&](int j, int m) {
    const uint32_t t = hb[j][m] + db[j];
    const bool wrap = t < db[j];  // carry out: raw + db >= p
    hb[j][m] = wrap ? t + kBias : t;  // on a carry t is the new raw hash itself
    const uint32_t cn = cb[j][m] + (wrap ? dc2[j] : dc1[j]);
    cb[j][m] = min(cn, cn - kr[j].c);  // cn < 2c: one subtraction, unsigned
  };
  // words per map row (rows padded to hrow bits, hrow a multiple of 64)
  const uint32_t hrow32 = (uint32_t)(hrow >> 5);
  for (int64_t base = base0; base < d; base += stride) {  // block-uniform
    // HEAVYMIX: the draws are loaded first, so their memory latency overlaps the lookups
    uint32_t fill[U];
#pragma unroll
    for (int m = 0; m < U; ++m) {
      const int64_t i = base + threadIdx.x + (int64_t)m * kPruneBlock;
      fill[m] = HM && i < d ? rnd[i] >> 1 : 0u;
    }
    // all U * R lookups first (independent), then the appends
    uint32_t cnt[U];
#pragma unroll
    for (int m = 0; m < U; ++m) {
      cnt[m] = 0u;
      if constexpr (MAP == kMapCoarse) {
        // a coarse bit covers its cells' heavy bits, so a coordinate with fewer than `need`
        // coarse-set rows is out without a global read; the others confirm their set rows in
        // the fine map (global reads, the cost here: L2 requests) while `need` is in reach
        Cell ev[R];
        uint32_t cset = 0u, nset = 0u;
#pragma unroll
        for (int j = 0; j < R; ++j) {
          const uint32_t col = cb[j][m];
          advance(j, m);
          ev[j] = (Cell)j * (Cell)hrow + col;
          const uint32_t cbit = ev[j] >> coarse_log2;
          const uint32_t bit = bit_at(sm[cbit >> 5], cbit);
          cset |= bit << j;
          nset += bit;
        }
        if (nset >= (uint32_t)need) {
          uint32_t left = nset;  // coarse-set rows not yet confirmed, this one included
#pragma unroll
          for (int j = 0; j < R; ++j) {
            if ((cset >> j) & 1u) {
              if (cnt[m] + left >= (uint32_t)need) cnt[m] += (heavy[ev[j] >> 5] >> (ev[j] & 31)) & 1u;
              --left;
            }
          }
        }
      } else if constexpr (MAP == kMapFine) {
#pragma unroll
        for (int j = 0; j < R; ++j) {
          const uint32_t col = cb[j][m];
          advance(j, m);
          cnt[m] += bit_at(sm[(uint32_t)j * hrow32 + (col >> 5)], col);
        }
      } else {
#pragma unroll
        for (int j = 0; j < R; ++j) {
          const uint32_t col = cb[j][m];
          advance(j, m);
          const Cell e = (Cell)j * (Cell)hrow + col;
          // global reads are the cost here (L2 requests): skip a row once the coordinate
          // cannot reach `need` with the rows left, which leaves the keep decision unchanged
          if (cnt[m] + (uint32_t)(R - j) >= (uint32_t)need) cnt[m] += (heavy[e >> 5] >> (e & 31)) & 1u;
        }
      }
    }
    // keep the lookups together, ahead of the appends (the compiler would otherwise sink
    // each coordinate's into its own guarded block and wait once per coordinate)
#pragma unroll
    for (int m = 0; m < U; ++m) asm volatile("" : "+v"(cnt[m]));
#pragma unroll
    for (int m = 0; m < U; ++m) {
      const int64_t i = base + threadIdx.x + (int64_t)m * kPruneBlock;
      bool keep = i < d && cnt[m] >= (uint32_t)need;
      if constexpr (HM) keep = keep || (i < d && fill[m] >= tau0);
      if (keep) {
        const uint32_t pos = atomicAdd(&bn, 1u);
        if (pos < (uint32_t)buf_cap) {
          buf[pos] = (uint32_t)i;
        } else {  // buffer full within this pass (dense survivors): queue directly
          queue[atomicAdd(&ctl->n_surv, 1u)] = (uint32_t)i;
        }
      }
      if (i < d && (i & 31) == 0) bitmap[i >> 5] = 0u;
    }
    __syncthreads();
    const uint32_t n = min(bn, (uint32_t)buf_cap);
    const bool last = base + stride >= d;
    if (n >= (uint32_t)(buf_cap / 2) || (last && n > 0)) {
      if (threadIdx.x == 0) gbase = atomicAdd(&ctl->n_surv, n);
      __syncthreads();
      const uint32_t g0 = gbase;
      for (uint32_t t = threadIdx.x; t < n; t += kPruneBlock) queue[g0 + t] = buf[t];
      __syncthreads();
      if (threadIdx.x == 0) bn = 0;
    }
    __syncthreads();
  }
}

// k_survivors: two blocks of 512 threads per CU (25.6M x 8: 15.8-16.1 us; one block of 256, 512
// or 1024 threads per CU: 18.8, 17.0, 18.8 us; four of 512: 17.9 us)
constexpr int kSurvBlock = 512;
constexpr int kSurvBuf = 2048;  // per-block LDS candidate buffer of k_survivors (at least 2 * kSurvBlock)

template <int R, bool HM>
__global__ void __launch_bounds__(kSurvBlock) k_survivors(HashSet hs, const float* __restrict__ merged,
                                                      SelectCtl* __restrict__ ctl, const uint32_t* __restrict__ queue,
                                                      uint32_t* __restrict__ cand_key, int32_t* __restrict__ cand_idx,
                                                      int64_t cap, const uint32_t* __restrict__ rnd,
                                                      uint32_t* __restrict__ hist_c) {
  __shared__ uint32_t bkey[kSurvBuf];
  __shared__ int32_t bidx[kSurvBuf];
  __shared__ uint32_t h[kDigit1Bins];
  __shared__ uint32_t bn, gbase, nheavy;
  for (int b = threadIdx.x; b < kDigit1Bins; b += kSurvBlock) h[b] = 0u;
  RowConst kr[R];
#pragma unroll
  for (int j = 0; j < R; ++j) kr[j] = row_const(hs, j);
  const uint32_t tau0 = ctl->tau0;
  const double theta = HM ? ctl->theta : 0.0;
  const int64_t n = ctl->n_surv;
  const int lane = threadIdx.x & 63;
  if (threadIdx.x == 0) {
    bn = 0u;
    nheavy = 0u;
  }
  __syncthreads();
  uint32_t mine = 0;
  const int64_t stride = (int64_t)gridDim.x * kSurvBlock;
  for (int64_t t0 = (int64_t)blockIdx.x * kSurvBlock; t0 < n; t0 += stride) {  // block-uniform trip count
    const int64_t t = t0 + threadIdx.x;
    bool cand = false;
    uint32_t key = 0u, i = 0u;
    if (t < n) {
      i = queue[t];
      const float e = estimate_val<R>(kr, merged, i);
      if constexpr (HM) {
        const bool hv = (double)e * (double)e >= theta;
        key = hv ? (0x80000000u | abs_key(e)) : (rnd[i] >> 1);
        cand = hv || key >= tau0;
        mine += hv ? 1u : 0u;
      } else {
        key = abs_key(e);
        cand = key >= tau0;
      }
    }
    hist_add(h, cand, key >> kDigit1Shift);
    // block-local append (one LDS atomic per wave); at most kSurvBlock per pass, so the buffer,
    // flushed whenever it is half full, never overflows
    const uint64_t bal = __ballot(cand);
    uint32_t wbase = 0u;
    if (lane == 0 && bal) wbase = atomicAdd(&bn, (uint32_t)__popcll(bal));
    wbase = __shfl(wbase, 0);
    if (cand) {
      const uint32_t pos = wbase + (uint32_t)__popcll(bal & ((1ull << lane) - 1ull));
      bkey[pos] = key;
      bidx[pos] = (int32_t)i;
    }
    __syncthreads();
    const uint32_t nb = bn;
    if (nb >= (uint32_t)(kSurvBuf / 2) || (t0 + stride >= n && nb > 0)) {
      if (threadIdx.x == 0) gbase = atomicAdd(&ctl->n_cand, nb);
      __syncthreads();
      const int64_t g0 = gbase;
      for (uint32_t u = threadIdx.x; u < nb; u += kSurvBlock) {
        if (g0 + u < cap) {
          cand_key[g0 + u] = bkey[u];
          cand_idx[g0 + u] = bidx[u];
        }
      }
      __syncthreads();
      if (threadIdx.x == 0) bn = 0u;
    }
    __syncthreads();
  }
  if constexpr (HM) {
    if (mine) atomicAdd(&nheavy, mine);
  }
  __syncthreads();
  if constexpr (HM) {
    if (threadIdx.x == 0 && nheavy) atomicAdd(&ctl->n_heavy, (unsigned long long)nheavy);
  }
  for (int b = threadIdx.x; b < kDigit1Bins; b += kSurvBlock) {
    const uint32_t c = h[b];
    if (c) atomicAdd(&hist_c[b], c);
  }
}

// ------------------------------------------------------------------------------------
// Step 5: bitmap -> ascending index list.

// Look-back word of emit block b: 0 until published, then kFlagAgg | (the block's own count),
// then kFlagIncl | (the count of blocks 0..b together). The count is all a word carries, so
// relaxed device-scope loads and stores of the word suffice (no fence orders other data).
constexpr unsigned long long kFlagAgg = 1ull << 62, kFlagIncl = 2ull << 62;
constexpr unsigned long long kFlagCount = 0xffffffffull;
// A block polls a window of predecessors' words at most spin_max times before it counts the
// bitmap words before its own directly (the blocks start in ticket order, so a predecessor is
// running and publishes without waiting on later blocks; the bound makes every wait finite
// regardless). spin_max < 0: every block counts directly.

__device__ __forceinline__ unsigned long long flag_load(const unsigned long long* p) {
  return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void flag_store(unsigned long long* p, unsigned long long v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Bitmap -> ascending index list in one pass. Block b (by ticket, i.e. in start order) owns
// words [b W, (b + 1) W): it counts its bits, publishes the count, adds the counts of the
// blocks before it (walking back until a block that has published its inclusive count),
// publishes its own inclusive count and writes its indices from that offset.
__global__ void __launch_bounds__(kSelBlock) k_emit(const uint32_t* __restrict__ bitmap, int64_t words,
                                                    SelectCtl* __restrict__ ctl,
                                                    unsigned long long* __restrict__ flags,
                                                    int32_t* __restrict__ idx, uint32_t k, int spin_max) {
  __shared__ uint32_t shw[kSelBlock / 64];
  __shared__ uint32_t sb, sexcl, sdirect;
  if (threadIdx.x == 0) {
    sb = atomicAdd(&ctl->emit_ticket, 1u);
    sdirect = 0u;
  }
  __syncthreads();
  const int64_t b = sb;
  const int64_t w0 = b * kEmitWordsPerBlock + (int64_t)threadIdx.x * kEmitWordsPerThread;
  uint32_t wv[kEmitWordsPerThread];
  uint32_t cnt = 0;
#pragma unroll
  for (int m = 0; m < kEmitWordsPerThread; ++m) {
    wv[m] = (w0 + m < words) ? bitmap[w0 + m] : 0u;
    cnt += __popc(wv[m]);
  }
  uint32_t total;
  const uint32_t incl = block_scan_incl<kSelBlock>(cnt, shw, total);
  if (threadIdx.x < 64) {  // the first wave publishes and looks back, 64 predecessors at a time
    const int lane = threadIdx.x;
    if (lane == 0) flag_store(&flags[b], (b == 0 ? kFlagIncl : kFlagAgg) | total);
    uint32_t excl = 0;
    bool direct = spin_max < 0 && b > 0;
    for (int64_t top = direct ? -1 : b - 1; top >= 0; top -= 64) {
      const int64_t j = top - lane;  // lane 0 is the nearest predecessor
      unsigned long long f = j >= 0 ? flag_load(&flags[j]) : kFlagIncl;  // before block 0: 0
      uint64_t incl_lanes, need;
      for (int spin = 0;; ++spin) {
        incl_lanes = __ballot((f & kFlagIncl) != 0ull);
        // lanes up to the nearest inclusive word must have published
        need = incl_lanes ? ((2ull << __builtin_ctzll(incl_lanes)) - 1ull) : ~0ull;
        if ((__ballot(f == 0ull) & need) == 0ull) break;
        if (spin >= spin_max) {
          direct = true;
          break;
        }
        __builtin_amdgcn_s_sleep(1);
        if (f == 0ull) f = flag_load(&flags[j]);
      }
      if (direct) break;
      uint32_t part = ((need >> lane) & 1ull) ? (uint32_t)(f & kFlagCount) : 0u;
#pragma unroll
      for (int o = 32; o > 0; o >>= 1) part += __shfl_xor(part, o, 64);
      excl += part;
      if (incl_lanes) break;
    }
    if (lane == 0) {
      sdirect = direct ? 1u : 0u;
      if (b > 0 && !direct) flag_store(&flags[b], kFlagIncl | (excl + total));
      sexcl = excl;
    }
  }
  __syncthreads();
  if (sdirect) {  // every word before this block's, counted by the whole block
    uint32_t before = 0;
    for (int64_t w = threadIdx.x; w < b * kEmitWordsPerBlock; w += kSelBlock) before += __popc(bitmap[w]);
    uint32_t all;
    (void)block_scan_incl<kSelBlock>(before, shw, all);
    if (threadIdx.x == 0) {
      sexcl = all;
      flag_store(&flags[b], kFlagIncl | (all + total));
    }
    __syncthreads();
  }
  uint32_t pos = sexcl + incl - cnt;
  const int64_t wb = b * kEmitWordsPerBlock + (int64_t)threadIdx.x * kEmitWordsPerThread;
#pragma unroll
  for (int m = 0; m < kEmitWordsPerThread; ++m) {
    uint32_t w = wv[m];
    while (w) {
      const int bit = __ffs(w) - 1;
      if (pos < k) idx[pos] = (int32_t)((wb + m) * 32 + bit);
      ++pos;
      w &= w - 1u;
    }
  }
}

// ------------------------------------------------------------------------------------
// HEAVYMIX as printed (Alg. 2). The l2-norm-squared estimate is the median over rows of
// sum_col S[j][col]^2 in fp64, each row summed in one fixed order (a pairwise tree over
// the squares padded with zeros to a power of two, adjacent pairs level by level), so the
// heavy test est_i^2 >= l2sq / k is a function of S alone. Keys then rank the heavy set
// above the fill: heavy i gets 0x80000000 | bits(|est_i|), the others their draw
// rnd[i] >> 1, and the radix selection above takes the k largest, ties to the lower index:
// all of H (or its k largest |est| when |H| >= k) plus the l = k - |H| non-heavy
// coordinates with the largest draws.

constexpr int kTreeLeaves = 2048;  // leaves per block of one tree pass (1024 threads)

// One tree pass: block b reduces the aligned group of G leaves (G a power of two, at most
// kTreeLeaves) of row j = b / (n / G) to one value, adding adjacent pairs level by level.
// First pass (sq != nullptr): leaf t of row j is sq[j][t]^2 for t < c, else 0 (n = padded
// width). Later passes: leaf t is in[j * n + t].
__global__ void __launch_bounds__(kTreeLeaves / 2) k_sq_tree(const float* __restrict__ sq,
                                                            const double* __restrict__ in, int64_t c, int64_t n,
                                                            int64_t G, double* __restrict__ out) {
  __shared__ double t2[kTreeLeaves / 2];
  const int64_t groups = n / G;
  const int64_t j = blockIdx.x / groups, base = (blockIdx.x - j * groups) * G;
  const int tid = threadIdx.x;
  auto leaf = [&](int64_t t) -> double {
    if (sq) {
      if (t >= c) return 0.0;
      const double x = (double)sq[j * c + t];
      return x * x;
    }
    return in[j * n + t];
  };
  if (G == 1) {
    if (tid == 0) out[blockIdx.x] = leaf(base);
    return;
  }
  int64_t w = G / 2;
  if (tid < w) t2[tid] = leaf(base + 2 * tid) + leaf(base + 2 * tid + 1);
  __syncthreads();
  for (; w > 1; w /= 2) {
    double a = 0.0;
    if (tid < w / 2) a = t2[2 * tid] + t2[2 * tid + 1];
    __syncthreads();
    if (tid < w / 2) t2[tid] = a;
    __syncthreads();
  }
  if (tid == 0) out[blockIdx.x] = t2[0];
}

// Median of the r row sums (insertion sort; even r: fl(fl(m1 + m2) * 0.5)), the threshold
// theta = l2sq / k, and the heavy counter reset. One thread.
__global__ void k_theta(const double* __restrict__ rows, int r, int64_t k, SelectCtl* __restrict__ ctl) {
  if (threadIdx.x != 0) return;
  double v[kMaxRows];
  for (int j = 0; j < r; ++j) v[j] = rows[j];
  for (int a = 1; a < r; ++a) {
    const double x = v[a];
    int b = a - 1;
    while (b >= 0 && v[b] > x) {
      v[b + 1] = v[b];
      --b;
    }
    v[b + 1] = x;
  }
  const double med = (r & 1) ? v[r / 2] : 0.5 * (v[r / 2 - 1] + v[r / 2]);
  ctl->l2sq = med;
  ctl->theta = med / (double)k;
  ctl->n_heavy = 0ull;
}

// Estimate + HEAVYMIX key + digit-1 histogram + |H|.
template <int R>
// gated: act only when the pruned pass raised the fallback flag; count_heavy: add |H| to
// ctl->n_heavy (off after a pruned pass, which already counted it).
__global__ void __launch_bounds__(kBlock) k_unsketch_hm(HashSet hs, const float* __restrict__ merged, int64_t d,
                                                        const uint32_t* __restrict__ rnd, float* __restrict__ est,
                                                        uint32_t* __restrict__ keys, uint32_t* __restrict__ hist,
                                                        uint32_t* __restrict__ bitmap, SelectCtl* __restrict__ ctl,
                                                        int gated, int count_heavy) {
  if (gated && !fallback_needed(ctl)) return;
  __shared__ uint32_t h[kDigit1Bins];
  __shared__ uint32_t nh;
  for (int b = threadIdx.x; b < kDigit1Bins; b += kBlock) h[b] = 0u;
  if (threadIdx.x == 0) nh = 0u;
  RowConst kr[R];
#pragma unroll
  for (int j = 0; j < R; ++j) kr[j] = row_const(hs, j);
  const double theta = ctl->theta;
  __syncthreads();
  uint32_t mine = 0;
  const int64_t stride = (int64_t)gridDim.x * kBlock;
  const int64_t i0 = (int64_t)blockIdx.x * kBlock + threadIdx.x;
  uint32_t hb[R], hsg[R], db[R], dsg[R];
#pragma unroll
  for (int j = 0; j < R; ++j) {
    hb[j] = mod_mersenne_affine(kr[j].a, kr[j].b, (uint32_t)i0);
    hsg[j] = mod_mersenne_affine(kr[j].a2, kr[j].b2, (uint32_t)i0);
    db[j] = mod_mersenne_affine(kr[j].a, 0u, (uint32_t)stride);
    dsg[j] = mod_mersenne_affine(kr[j].a2, 0u, (uint32_t)stride);
  }
  for (int64_t i = i0; i < d; i += stride) {
    float val[R];
#pragma unroll
    for (int j = 0; j < R; ++j) {
      const uint32_t col = mod_c(hb[j], kr[j].c, kr[j].magic, kr[j].shift);
      val[j] = apply_sign(merged[(int64_t)j * hs.c + col], sign_flip_of(hsg[j]));
      hb[j] = add_mod_mersenne(hb[j], db[j]);
      hsg[j] = add_mod_mersenne(hsg[j], dsg[j]);
    }
    sort_net<R>(val);
    const float e = median_sorted<R>(val);
    if (est) est[i] = e;
    const double ed = (double)e;
    const bool heavy = ed * ed >= theta;
    const uint32_t key = heavy ? (0x80000000u | abs_key(e)) : (rnd[i] >> 1);
    mine += heavy ? 1u : 0u;
    keys[i] = key;
    atomicAdd(&h[key >> kDigit1Shift], 1u);
    if ((i & 31) == 0) bitmap[i >> 5] = 0u;
  }
  if (mine) atomicAdd(&nh, mine);
  __syncthreads();
  for (int b = threadIdx.x; b < kDigit1Bins; b += kBlock) {
    const uint32_t n = h[b];
    if (n) atomicAdd(&hist[b], n);
  }
  if (count_heavy && threadIdx.x == 0 && nh) atomicAdd(&ctl->n_heavy, (unsigned long long)nh);
}

__global__ void k_hm_out(const SelectCtl* __restrict__ ctl, int64_t* __restrict__ n_heavy, double* __restrict__ l2sq) {
  if (threadIdx.x != 0) return;
  if (n_heavy) *n_heavy = (int64_t)ctl->n_heavy;
  if (l2sq) *l2sq = ctl->l2sq;
}

template <int R>
void launch_unsketch_r(const HashSet& hs, int64_t d, int num_cus, const SelectBufs& b, hipStream_t s,
                       const float* merged, float* est, SelectCtl* gate) {
  if (d <= (int64_t)kUnsketchSmall * kBlock * num_cus)
    hipLaunchKernelGGL((k_unsketch<R, 2>), dim3(grid_for(d, 2 * kBlock, num_cus)), dim3(kBlock), 0, s, hs, merged, d,
                       est, b.cand_key, b.hist, b.bitmap, gate);
  else
    hipLaunchKernelGGL((k_unsketch<R, 1>), dim3(grid_for(d, kBlock, 4 * num_cus)), dim3(kBlock), 0, s, hs, merged, d,
                       est, b.cand_key, b.hist, b.bitmap, gate);
}

template <int R, bool HM>
void launch_prune_r(gs_ctx* x, hipStream_t s, const float* merged, int64_t k, const uint32_t* rnd) {
  const int M = (int)(x->d < kSampleMax ? x->d : kSampleMax);
  const double mk = (double)M * (double)k / (double)x->d;
  // expected sampled keys above the k-th key: mk (sd ~ sqrt(mk)); the margin is ~8 sd
  double rho_d = std::ceil(1.2 * mk + 5.0 * std::sqrt(mk) + 8.0);
  if (rho_d > M) rho_d = M;
  if (rho_d < 1) rho_d = 1;
  hipLaunchKernelGGL((k_sample<R, HM>), dim3((M + kBlock - 1) / kBlock), dim3(kBlock), 0, s, x->hs, merged, x->d, M,
                     rnd, x->sample_keys, x->hist_s);
  const int64_t nbits = (int64_t)x->r * x->heavy_row;  // heavy-cell map bits (padded rows)
  hipLaunchKernelGGL(k_heavy, dim3(grid_for(nbits, kSelBlock * kHeavyUnroll, x->num_cus)), dim3(kSelBlock), 0, s,
                     merged, x->c, x->heavy_row, x->r, x->ctl, x->heavy, HM ? 1 : 0, x->sample_keys, M,
                     (uint32_t)rho_d, (uint32_t)k, x->hist_s);
  // with the bitmap in LDS one block fits a CU: launch one per CU so the map is loaded once
  const int pgrid = grid_for(x->d, 4 * kPruneBlock, x->prune_map_in_lds ? x->num_cus : 2 * x->num_cus);
  const dim3 pb(kPruneBlock);
  if (!x->prune_map_in_lds) {
    hipLaunchKernelGGL((k_pruned<R, HM, kMapGlobal>), dim3(pgrid), pb, 0, s, x->hs, x->d, x->ctl,
                       x->heavy, x->heavy, x->prune_map_words, x->heavy_row, 0, x->prune_buf_cap, x->keys,
                       x->bitmap, rnd, x->hist_s);
  } else if (x->prune_coarse_log2 > 0) {
    hipLaunchKernelGGL(k_coarse, dim3(grid_for(x->prune_coarse_words, kBlock, 4 * x->num_cus)), dim3(kBlock), 0, s,
                       x->heavy, nbits / 32, x->prune_coarse_log2, x->coarse, x->prune_coarse_words);
    hipLaunchKernelGGL((k_pruned<R, HM, kMapCoarse>), dim3(pgrid), pb, 0, s, x->hs, x->d, x->ctl,
                       x->heavy, x->coarse, x->prune_map_words, x->heavy_row, x->prune_coarse_log2,
                       x->prune_buf_cap, x->keys,
                       x->bitmap, rnd, x->hist_s);
  } else {
    hipLaunchKernelGGL((k_pruned<R, HM, kMapFine>), dim3(pgrid), pb, 0, s, x->hs, x->d, x->ctl,
                       x->heavy, x->heavy, x->prune_map_words, x->heavy_row, 0, x->prune_buf_cap, x->keys,
                       x->bitmap, rnd, x->hist_s);
  }
  hipLaunchKernelGGL((k_survivors<R, HM>), dim3(2 * x->num_cus), dim3(kSurvBlock), 0, s, x->hs, merged, x->ctl, x->keys,
                     x->cand_key, x->cand_idx, x->cand_cap, rnd, x->hist_c);
}

// digit2 -> select2 -> mark -> emit over the candidates: the pruned pass's (pruned = 1,
// unless it fell short of k) or the full estimate's dense ones.
hipError_t launch_select_tail(int64_t d, int num_cus, const SelectBufs& b, hipStream_t s, int64_t k, int pruned,
                              int32_t* idx) {
  // one block (of 1,024 threads) per four CUs for the pruned candidates (a few times k: fewer
  // blocks each append their staged keys and histogram with fewer atomics that queue at the
  // same addresses); the full estimate's dense ones (d) get up to 8 * (CUs) blocks (a pruned
  // pass's fallback keeps the smaller grid)
  int g2 = std::max(1, num_cus / 4);
  if (!pruned) g2 = std::max(g2, grid_for(d, 8192, 8 * num_cus));
  hipLaunchKernelGGL(k_digit2, dim3(g2), dim3(kDigit2Block), 0, s, b.cand_key, b.cand_idx, b.ctl, b.cand_cap, d, b.hist_c,
                     b.hist, pruned, (uint32_t)k, b.hist2, b.keys, b.stage_idx, b.bitmap);
  hipLaunchKernelGGL(k_select2, dim3(1), dim3(kSelBlock), 0, s, b.ctl, b.hist2, b.keys, b.stage_idx, b.hist_c, b.hist,
                     pruned, (uint32_t)k, b.emit_flags, b.emit_blocks);
  hipLaunchKernelGGL(k_mark, dim3(num_cus), dim3(kBlock), 0, s, b.keys, b.stage_idx, b.ctl, b.bitmap);
  const int64_t words = (d + 31) / 32;
  hipLaunchKernelGGL(k_emit, dim3((unsigned)b.emit_blocks), dim3(kSelBlock), 0, s, b.bitmap, words, b.ctl,
                     b.emit_flags, idx, (uint32_t)k, b.emit_spin);
  return hipGetLastError();
}

hipError_t launch_select_tail(gs_ctx* x, hipStream_t s, int64_t k, int pruned, int32_t* idx) {
  return launch_select_tail(x->d, x->num_cus, select_bufs(x), s, k, pruned, idx);
}

}  // namespace

int64_t emit_blocks_for(int64_t d) {
  const int64_t words = (d + 31) / 32;
  return (words + kEmitWordsPerBlock - 1) / kEmitWordsPerBlock;
}

hipError_t prepare_prune(gs_ctx* x) {
  const int64_t rc = (int64_t)x->r * x->heavy_row;  // bits of the heavy-cell map (padded rows)
  const int64_t words = rc / 32;
  const int64_t lds_max = 160 * 1024 - 256;
  // the fine map in LDS if it fits beside a 512-entry queue buffer; else the coarsest-needed
  // coarse map (2 .. 32 cells per bit); else the fine map from global memory
  int64_t map_words = words;
  int log2g = 0;
  while ((lds_max - map_words * 4) / 4 < 512 && log2g < 5) {
    ++log2g;
    map_words = (rc + (32ll << log2g) - 1) / (32ll << log2g);
    map_words += map_words & 1;
  }
  int64_t buf = (lds_max - map_words * 4) / 4;
  if (buf > 8192) buf = 8192;
  if (buf >= 512) {
    x->prune_map_in_lds = 1;
    x->prune_coarse_log2 = log2g;
    x->prune_map_words = map_words;
    x->prune_buf_cap = (int)buf;
    if (log2g > 0) {
      x->prune_coarse_words = map_words;
      const hipError_t e = hipMalloc(reinterpret_cast<void**>(&x->coarse), (size_t)map_words * sizeof(uint32_t));
      if (e != hipSuccess) return e;
    }
  } else {
    x->prune_map_in_lds = 0;
    x->prune_coarse_log2 = 0;
    x->prune_map_words = words;
    x->prune_buf_cap = 8192;
  }
  // the map (when in LDS), the queue buffer and two counters share the pass's LDS array
  if ((x->prune_map_in_lds ? x->prune_map_words : 0) + x->prune_buf_cap + 2 > kPruneLdsWords)
    return hipErrorInvalidValue;
  return hipSuccess;
}

hipError_t launch_unsketch_topk(gs_ctx* x, hipStream_t s, const float* merged, int64_t k, float* est, int32_t* idx) {
  // With an estimate vector requested, or a sketch small enough (d*r at most
  // prune_min_cells) that the full estimate is the cheaper chain, every coordinate is
  // estimated. Otherwise the pruned path runs and the full estimate only acts if the pruned
  // candidates fell short of k.
  const bool prune = est == nullptr && x->d * x->r > x->prune_min_cells;
  SelectCtl* gate = prune ? x->ctl : nullptr;
  switch (x->r) {
#define GS_R_CASE(RR) \
  case RR:                                            \
    if (prune) launch_prune_r<RR, false>(x, s, merged, k, nullptr);  \
    launch_unsketch_r<RR>(x->hs, x->d, x->num_cus, select_bufs(x), s, merged, est, gate);  \
    break;
    GS_R_CASE(1) GS_R_CASE(2) GS_R_CASE(3) GS_R_CASE(4) GS_R_CASE(5) GS_R_CASE(6) GS_R_CASE(7) GS_R_CASE(8)
    GS_R_CASE(9) GS_R_CASE(10) GS_R_CASE(11) GS_R_CASE(12) GS_R_CASE(13) GS_R_CASE(14) GS_R_CASE(15) GS_R_CASE(16)
#undef GS_R_CASE
    default: return hipErrorInvalidValue;
  }
  return launch_select_tail(x, s, k, prune ? 1 : 0, idx);
}

hipError_t launch_unsketch_topk_dense(const HashSet& hs, int64_t d, int num_cus, const SelectBufs& b, hipStream_t s,
                                      const float* merged, int64_t k, float* est, int32_t* idx) {
  switch (hs.r) {
#define GS_R_CASE(RR) \
  case RR: launch_unsketch_r<RR>(hs, d, num_cus, b, s, merged, est, nullptr); break;
    GS_R_CASE(1) GS_R_CASE(2) GS_R_CASE(3) GS_R_CASE(4) GS_R_CASE(5) GS_R_CASE(6) GS_R_CASE(7) GS_R_CASE(8)
    GS_R_CASE(9) GS_R_CASE(10) GS_R_CASE(11) GS_R_CASE(12) GS_R_CASE(13) GS_R_CASE(14) GS_R_CASE(15) GS_R_CASE(16)
#undef GS_R_CASE
    default: return hipErrorInvalidValue;
  }
  return launch_select_tail(d, num_cus, b, s, k, 0, idx);
}

hipError_t launch_heavymix_topk(gs_ctx* x, hipStream_t s, const float* merged, int64_t k, const uint32_t* rnd,
                                float* est, int32_t* idx, int64_t* n_heavy, double* l2sq) {
  // row sums of squares, pass by pass (each reduces aligned groups of up to 2048 values)
  const int64_t npad = l2_pad(x->c);
  int64_t n = npad;
  const double* in = nullptr;
  double* out = x->l2buf;
  bool first = true;
  while (first || n > 1) {
    const int64_t G = n < kTreeLeaves ? n : kTreeLeaves;
    const int64_t groups = n / G;
    hipLaunchKernelGGL(k_sq_tree, dim3((unsigned)(x->r * groups)), dim3(kTreeLeaves / 2), 0, s,
                       first ? merged : nullptr, in, x->c, n, G, out);
    in = out;
    out = (out == x->l2buf) ? x->l2buf + x->l2_half : x->l2buf;
    n = groups;
    first = false;
  }
  hipLaunchKernelGGL(k_theta, dim3(1), dim3(64), 0, s, in, x->r, k, x->ctl);
  // As in launch_unsketch_topk: the full estimate with an estimate vector or a small sketch,
  // else the pruned pass, with the full one acting only if its candidates fell short of k.
  const bool prune = est == nullptr && x->d * x->r > x->prune_min_cells;
  switch (x->r) {
#define GS_R_CASE(RR)                                                                                              \
  case RR:                                                                                                         \
    if (prune) launch_prune_r<RR, true>(x, s, merged, k, rnd);                                                     \
    hipLaunchKernelGGL(k_unsketch_hm<RR>, dim3(grid_for(x->d, kBlock, 4 * x->num_cus)), dim3(kBlock), 0, s, x->hs, \
                       merged, x->d, rnd, est, x->cand_key, x->hist, x->bitmap, x->ctl, prune ? 1 : 0,            \
                       prune ? 0 : 1);                                                                             \
    break;
    GS_R_CASE(1) GS_R_CASE(2) GS_R_CASE(3) GS_R_CASE(4) GS_R_CASE(5) GS_R_CASE(6) GS_R_CASE(7) GS_R_CASE(8)
    GS_R_CASE(9) GS_R_CASE(10) GS_R_CASE(11) GS_R_CASE(12) GS_R_CASE(13) GS_R_CASE(14) GS_R_CASE(15) GS_R_CASE(16)
#undef GS_R_CASE
    default: return hipErrorInvalidValue;
  }
  if (n_heavy || l2sq) hipLaunchKernelGGL(k_hm_out, dim3(1), dim3(64), 0, s, x->ctl, n_heavy, l2sq);
  return launch_select_tail(x, s, k, prune ? 1 : 0, idx);
}

int64_t l2_pad(int64_t c) {
  int64_t n = 1;
  while (n < c) n *= 2;
  return n;
}

}  // namespace gs