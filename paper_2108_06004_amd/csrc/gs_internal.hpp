// gs_internal.hpp -- host-side context and kernel launchers shared by the library's
// translation units. Not part of the public ABI (include/gs.h is).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <string>

#include "../../include/gs.h"
#include "gs_device.hpp"

// Top-k selection works on 32-bit keys (the bits of |estimate|) in three radix digits.
namespace gs {
constexpr int kDigit1Shift = 20;  // digit 1: key bits 31..20 (12 bits; |est| keys leave bit 31 clear,
constexpr int kDigit1Bins = 4096; // HEAVYMIX keys use it to rank the heavy set above the fill)
constexpr int kDigitBins = 1024;  // digits 2 and 3: key bits 19..10 and 9..0

// Device-resident control block of the selection (one per context).
struct SelectCtl {
  uint32_t k;           // number to select
  uint32_t b1;          // digit-1 bucket holding the k-th key
  uint32_t above1;      // keys in digit-1 buckets above b1
  uint32_t n_cand;      // candidates appended by the pruned pass (dense candidates: d)
  uint32_t tau;         // the k-th largest key
  uint32_t iota;        // largest index taken among keys equal to tau
  uint32_t tau0;        // pruning bound: a key no larger than the k-th key (when no fallback)
  uint32_t fallback;    // 1: fewer than k coordinates reach tau0, run the unpruned selection
  uint32_t n_surv;      // coordinates queued by the pruned pass for an exact estimate
  double l2sq;          // HEAVYMIX: l2-norm-squared estimate (median of the pairwise row sums)
  double theta;         // HEAVYMIX: heavy threshold l2sq / k
  unsigned long long n_heavy;  // HEAVYMIX: |H|
  uint32_t n_stage2;    // keys of the digit-1 bucket b1 staged for the digit-3 pass
  uint32_t n_staged;    // n_stage2 as k_select2 found it, for the emit (n_stage2 is reset there)
  uint32_t emit_ticket; // order in which the emit's workgroups start (their look-back order)
};
// Buffers of the dense selection (every coordinate a candidate) and of its radix tail: the
// context's scratch for gs_unsketch_topk and friends, or the static scratch of
// gs_unsketch_topk_static. hist, hist2, hist_c and ctl->n_stage2 are zero between calls.
struct SelectBufs {
  uint32_t* cand_key;   // [cand_cap] candidate keys (dense: key of coordinate t at t)
  int32_t* cand_idx;    // [cand_cap] candidate coordinates (read only for pruned candidates)
  int64_t cand_cap;
  uint32_t* keys;       // [d] staged keys of the digit-1 bucket of the k-th key
  int32_t* stage_idx;   // [d] their coordinates
  uint32_t* hist;       // [kDigit1Bins] digit-1 histogram of the dense keys
  uint32_t* hist2;      // [kDigitBins]
  uint32_t* hist_c;     // [kDigit1Bins] digit-1 histogram of pruned candidates
  SelectCtl* ctl;
  uint32_t* bitmap;     // [ceil(d/32)] output bitmap
  unsigned long long* emit_flags;  // [emit_blocks] look-back words of the emit (zero before it)
  int64_t emit_blocks;
  int emit_spin;        // polls of the emit's look-back before counting directly (< 0: never look back)
};
constexpr int kEmitSpinDefault = 1 << 20;
constexpr int kSampleMax = 16384;  // sampled estimates for the pruning bound
constexpr int64_t kPruneMinCells = 2000000;  // d*r below which the full estimate is faster (measured)

// Geometry of the gather-based sketch: tiles of W columns of one row, all P workers, fp64.
// The columns of row j are taken in the order of their scaled position t = theta_j * col
// mod c (theta_j coprime to c, so this is a permutation of the columns), and tile k of the
// row holds the columns with t in [k W, (k + 1) W). The bucket hash is affine, so
// consecutive coordinates' columns differ by one of two constants (a_j mod c, or that less
// p mod c when the raw hash wraps past p); theta_j is chosen to make both steps small in t,
// so consecutive coordinates mostly share a tile and a 128-byte line of the state mostly
// feeds one tile per row.
struct PullPlan {
  int32_t P, PP;          // workers; vI row length (P rounded up to a multiple of 4)
  int32_t W;              // columns per tile
  int32_t tiles_per_row;  // ceil(c / W)
  int32_t T;              // r * tiles_per_row
  int32_t S;              // list segments per tile (work items = T * S)
  int32_t NB;             // build chunks
  int32_t slots;          // resident pull workgroups (one per CU): the size of a round
  int64_t chunk;          // coordinates per build chunk
  uint32_t theta[kMaxRows];      // column scaling of row j
  uint32_t theta_inv[kMaxRows];  // its inverse modulo c (position t -> column)
  // Packed lists: each tile's list starts at a multiple of kListGroup entries; an entry is
  // one word, the coordinate's offset from its group's base (the group's first coordinate)
  // in the low off_bits bits, the position in the tile above it, the sign in bit 31. When a
  // group's coordinates span too much for off_bits (or P > 16) the lists stay unpacked:
  // coordinates in `list`, position | sign << 15 in `codes`.
  int32_t packed;
  int32_t off_bits;
  // list build: t / W as (t * w_magic) >> w_shift, 1 / c, bits of a tile index
  uint32_t w_magic, w_shift;
  double inv_c;
  int32_t tile_bits;
  // LDS cell of position t in row j's tiles: t ^ ((t >> swz[j]) & 31) when swz[j] > 0, else t
  // (see tile_cell); a worker's column of cells is W rounded up to 32, plus 6, long.
  int32_t swz[kMaxRows];
};
constexpr int kListGroup = 64;
constexpr int64_t kMaxFillLds = 160 * 1024;  // LDS of the list-fill kernel holds T cursors

// Where element (worker q, coordinate i) of a per-worker array lives: q*qs + i*is.
// [P][d] (worker-major) is {d, 1}; the interleaved state [d][PP] is {1, PP}.
struct StateView {
  int64_t qs, is;
  __host__ __device__ int64_t at(int q, int64_t i) const { return (int64_t)q * qs + i * is; }
};
constexpr int kTilesPerCu = 1;               // resident pull workgroups per CU (LDS-limited)
}  // namespace gs

struct gs_ctx {
  int device = 0;
  int64_t d = 0, c = 0, k_max = 0;
  int32_t P = 0, r = 0;
  float rho = 0.f;
  int32_t reset_momentum = 1;
  int32_t state_layout = 0;   // GS_STATE_WORKER_MAJOR or GS_STATE_INTERLEAVED (u and v)
  int32_t state_stride = 0;   // row length of the interleaved state: P rounded up to a multiple of 4
  gs::HashSet hs{};
  int num_cus = 256;

  // scratch (device)
  uint32_t* keys = nullptr;       // [d] survivor queue of the pruned pass, then the staged keys
  uint32_t* hist = nullptr;       // [kDigit1Bins], zero between calls
  uint32_t* hist2 = nullptr;      // [kDigitBins] digit-2 histogram of bucket b1, zero between calls
  uint32_t* hist_s = nullptr;     // [kDigit1Bins] digit-1 histogram of the sampled keys, zero between calls
  uint32_t* hist_c = nullptr;     // [kDigit1Bins] digit-1 histogram of the pruned candidates, zero between calls
  gs::SelectCtl* ctl = nullptr;   // [1]
  int32_t* stage_idx = nullptr;   // [d] coordinates of the keys staged in `keys` for the digit-3 pass
  uint32_t* cand_key = nullptr;   // [cand_cap]
  int32_t* cand_idx = nullptr;    // [cand_cap]
  int64_t cand_cap = 0;
  uint32_t* bitmap = nullptr;     // [ceil(d/32)]
  unsigned long long* emit_flags = nullptr;  // [emit blocks] look-back words of the emit
  uint32_t* sample_keys = nullptr;  // [kSampleMax]
  uint32_t* heavy = nullptr;        // [r * heavy_row / 32] heavy-cell bitmap, rows padded to heavy_row bits
  int64_t heavy_row = 0;            // c rounded up to a multiple of 64: bit j * heavy_row + col is cell (j, col)
  int64_t prune_map_words = 0;      // words of the heavy bitmap
  int prune_map_in_lds = 0;         // 1: the pruned pass keeps a bitmap in LDS (fine, or coarse below)
  int prune_coarse_log2 = 0;        // > 0: LDS holds the coarse map, one bit per 2^this cells
  uint32_t* coarse = nullptr;       // coarse heavy-cell map (bit = OR of its cells' heavy bits)
  int64_t prune_coarse_words = 0;
  int prune_buf_cap = 0;            // LDS candidate buffer entries of the pruned pass
  int64_t emit_blocks = 0;
  int emit_spin = gs::kEmitSpinDefault;  // diagnostic override: GS_EMIT_SPIN
  // selections without an estimate vector prune when d*r exceeds this (0: always); below it
  // the full estimate takes fewer launches than the pruned pass's chain
  int64_t prune_min_cells = 0;
  // gather-based sketch (used when the plan fits; otherwise fp64 atomics into acc64)
  bool use_pull = false;
  gs::PullPlan plan{};
  uint32_t* list = nullptr;       // [list_cap] coordinates of each tile, ascending (or packed entries)
  uint16_t* codes = nullptr;      // [list_cap] unpacked lists: position in the tile | sign << 15
  uint32_t* bases = nullptr;      // [list_cap / kListGroup] packed lists: first coordinate of each group
  int64_t list_cap = 0;           // r*d + kListGroup*T (tiles start at multiples of kListGroup)
  int64_t* tile_off = nullptr;    // [T+1] tile starts in the list
  uint32_t* tile_n = nullptr;     // [T] entries of each tile
  float* vI = nullptr;            // [d][PP] worker-interleaved accumulators
  double* partial = nullptr;      // [S][r][c][P] fp64 tile sums
  double* acc64 = nullptr;        // [P][r][c] fp64 cell accumulators of the atomic path
  // HEAVYMIX row sums of squares: two ping-pong buffers of tree-pass results
  double* l2buf = nullptr;        // [2][l2_half]
  int64_t l2_half = 0;            // r * max(1, npad / 2048) with npad = next power of two >= c

  // stage timing of the fused steps (gs_timing_start / gs_timing_stop): events recorded on
  // the step's stream before the first stage and after each stage, for up to t_max steps
  bool timing = false;
  int32_t t_max = 0, t_step = 0;
  hipEvent_t* t_events = nullptr;  // [t_max][GS_STAGE_MARKS]

  std::string last_error;
};

namespace gs {
// The view of the caller's u and v (per the context's state layout), and of a [P][d] array.
inline StateView state_view(const gs_ctx* x) {
  return x->state_layout == GS_STATE_INTERLEAVED ? StateView{1, x->state_stride} : StateView{x->d, 1};
}
inline StateView worker_major_view(const gs_ctx* x) { return StateView{x->d, 1}; }
inline SelectBufs select_bufs(const gs_ctx* x) {
  return SelectBufs{x->cand_key, x->cand_idx, x->cand_cap, x->keys,   x->stage_idx, x->hist,
                    x->hist2,    x->hist_c,   x->ctl,      x->bitmap, x->emit_flags, x->emit_blocks,
                    x->emit_spin};
}

constexpr int kStageMarks = 6;  // events per timed step: before stage 0, after stages 0..4
// Record timing mark t (0..5) of the current step on `s` when timing is active; mark 5
// completes the step.
void stage_mark(gs_ctx* x, hipStream_t s, int t);
// Launchers (each enqueues on `s` and returns hipGetLastError()).
hipError_t launch_accumulate(const gs_ctx* x, hipStream_t s, const float* g, float* u, float* v);
hipError_t launch_fill_zero(hipStream_t s, float* p, int64_t n);
hipError_t launch_sketch_acc(const gs_ctx* x, hipStream_t s, const float* v, StateView sv);
hipError_t launch_sketch(const gs_ctx* x, hipStream_t s, const float* v, StateView sv, float* tables);
hipError_t launch_merge_acc(const gs_ctx* x, hipStream_t s, float* merged);
hipError_t launch_merge(const gs_ctx* x, hipStream_t s, const float* tables, float* merged);
hipError_t launch_unsketch_topk(gs_ctx* x, hipStream_t s, const float* merged, int64_t k, float* est, int32_t* idx);
hipError_t launch_heavymix_topk(gs_ctx* x, hipStream_t s, const float* merged, int64_t k, const uint32_t* rnd,
                                float* est, int32_t* idx, int64_t* n_heavy, double* l2sq);
int64_t l2_pad(int64_t c);
hipError_t launch_apply_update(const gs_ctx* x, hipStream_t s, const int32_t* idx, const float* values, int64_t k,
                               float lr, float* w);
hipError_t launch_sketch_state(gs_ctx* x, hipStream_t s, const float* merged, float* U, float* E, int64_t k,
                               int32_t* idx, float* values);
hipError_t launch_gather_reset(const gs_ctx* x, hipStream_t s, const int32_t* idx, int64_t k, float* u, float* v,
                               float* values);
int64_t emit_blocks_for(int64_t d);
// The estimate of every coordinate and the top-k over them (the full path of
// launch_unsketch_topk) on explicit buffers; r = hs.r, 1 <= k <= d.
hipError_t launch_unsketch_topk_dense(const HashSet& hs, int64_t d, int num_cus, const SelectBufs& b, hipStream_t s,
                                      const float* merged, int64_t k, float* est, int32_t* idx);
// Granlund-Montgomery reciprocal of the bucket modulus c (sets hs.c, hs.magic, hs.shift).
void set_divisor(HashSet& hs, uint32_t c);
// Message of the last failing context-free call on this thread (gs_create,
// gs_unsketch_topk_static), returned by gs_last_error(NULL); no heap allocation.
void set_free_error(const char* msg);
hipError_t prepare_prune(gs_ctx* x);
PullPlan make_pull_plan(const HashSet& hs, int64_t d, int32_t P, int32_t r, int64_t c, int num_cus);
hipError_t build_pull_lists(gs_ctx* x);
hipError_t launch_accumulate_vi(const gs_ctx* x, hipStream_t s, const float* g, float* u, float* v);
hipError_t launch_interleave(const gs_ctx* x, hipStream_t s, const float* v);
// The pull gathers rows of PP floats (16-byte aligned) from `rows`: the context's interleaved
// copy x->vI, or the caller's v itself when the state is interleaved. When pull_merges(x)
// (P <= 16 and one list segment per tile) it also writes the per-worker tables and/or the
// merged sketch (non-null outputs) and launch_merge_partials has nothing left to do; pass
// the same outputs to both.
hipError_t launch_pull(const gs_ctx* x, hipStream_t s, const float* rows, float* merged, float* tables);
// One worker (P = 1): the pull gathers the plain vector v[d] (4 bytes per coordinate), with
// no interleaved copy; the worker-major state of one worker is such a vector.
hipError_t launch_pull_flat(const gs_ctx* x, hipStream_t s, const float* v, float* merged, float* tables);
// A worker-major state with one worker is gathered directly (no interleaved copy).
inline bool flat_state(const gs_ctx* x) { return x->P == 1 && x->state_layout == GS_STATE_WORKER_MAJOR; }
bool pull_merges(const gs_ctx* x);
// Rows for the pull from the caller's state array v (GS_STATE_INTERLEAVED): v itself when it
// is 16-byte aligned, otherwise a copy enqueued into x->vI.
const float* pull_rows_of_state(const gs_ctx* x, hipStream_t s, const float* v, hipError_t* e);
hipError_t launch_merge_partials(const gs_ctx* x, hipStream_t s, float* merged, float* tables);
}  // namespace gs
