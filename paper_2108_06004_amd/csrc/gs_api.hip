// gs_api.hip -- the C ABI declared in include/gs.h: argument validation, the context and
// its device scratch, and the kernel sequence of each call.
#include <cmath>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <new>
#include <string>

#include "../../include/gs.h"
#include "gs_internal.hpp"

namespace {

// message of the last failing context-free call on this thread (gs_create,
// gs_unsketch_topk_static): a fixed buffer, so that setting it allocates nothing
thread_local char g_free_error[512];

constexpr int64_t kP = GS_MERSENNE_P;

gs_status fail(gs_ctx* x, gs_status st, const std::string& msg) {
  if (x) x->last_error = msg;
  return st;
}

gs_status device_status(gs_ctx* x, hipError_t e, const char* where) {
  if (e == hipSuccess) return GS_OK;
  return fail(x, GS_ERR_DEVICE, std::string(where) + ": " + hipGetErrorString(e));
}

template <typename T>
hipError_t alloc(T** p, int64_t count) {
  *p = nullptr;
  if (count <= 0) count = 1;
  return hipMalloc(reinterpret_cast<void**>(p), (size_t)count * sizeof(T));
}

void free_scratch(gs_ctx* x) {
  void* ptrs[] = {x->keys,     x->hist,     x->hist2,       x->hist_s, x->hist_c, x->ctl,     x->stage_idx,
                  x->cand_key, x->cand_idx, x->bitmap,      x->emit_flags, x->acc64, x->list,  x->codes,
                  x->bases,    x->tile_off, x->tile_n,      x->vI,     x->partial, x->sample_keys,
                  x->heavy,    x->l2buf,    x->coarse};
  for (void* p : ptrs)
    if (p) (void)hipFree(p);
  x->keys = nullptr;
  x->hist = nullptr;
  x->hist2 = nullptr;
  x->hist_s = nullptr;
  x->hist_c = nullptr;
  x->ctl = nullptr;
  x->stage_idx = nullptr;
  x->cand_key = nullptr;
  x->cand_idx = nullptr;
  x->bitmap = nullptr;
  x->emit_flags = nullptr;
  x->acc64 = nullptr;
  x->list = nullptr;
  x->codes = nullptr;
  x->bases = nullptr;
  x->tile_off = nullptr;
  x->tile_n = nullptr;
  x->vI = nullptr;
  x->partial = nullptr;
  x->sample_keys = nullptr;
  x->heavy = nullptr;
  x->l2buf = nullptr;
  x->coarse = nullptr;
}

bool valid_ab(const uint32_t* a, const uint32_t* b, int r) {
  for (int j = 0; j < r; ++j)
    if (a[j] < 1 || (int64_t)a[j] >= kP || (int64_t)b[j] >= kP) return false;
  return true;
}

hipStream_t as_stream(void* s) { return reinterpret_cast<hipStream_t>(s); }

// An interleaved v the pull cannot gather directly (16-byte pieces of its rows) goes through
// the context's interleaved copy, which an interleaved context has only with GS_OPT_ROW_COPY.
bool unaligned_without_copy(const gs_ctx* x, const float* v) {
  return x->use_pull && x->state_layout == GS_STATE_INTERLEAVED && x->P <= 16 && ((uintptr_t)v & 15u) != 0 &&
         x->vI == nullptr;
}
constexpr const char* kUnalignedMsg =
    ": interleaved v is not 16-byte aligned and the context has no row copy (GS_OPT_ROW_COPY)";

}  // namespace

namespace gs {
// Granlund-Montgomery reciprocal for 31-bit dividends: l = ceil(log2 c), m = ceil(2^(31+l)/c)
// (m < 2^32; for c = 1, l = 0 and m = 2^31), and floor(x / c) = floor(x * m / 2^(31+l)).
void set_divisor(HashSet& hs, uint32_t c) {
  uint32_t l = 0;
  while ((1ull << l) < c) ++l;
  const uint64_t num = 1ull << (31 + l);
  hs.c = c;
  hs.magic = (uint32_t)((num + c - 1) / c);
  hs.shift = 31 + l;
}

void set_free_error(const char* msg) { std::snprintf(g_free_error, sizeof g_free_error, "%s", msg ? msg : ""); }

void stage_mark(gs_ctx* x, hipStream_t s, int t) {
  if (!x->timing || x->t_step >= x->t_max) return;
  (void)hipEventRecord(x->t_events[(int64_t)x->t_step * kStageMarks + t], s);
  if (t == kStageMarks - 1) ++x->t_step;
}
}  // namespace gs

extern "C" {

const char* gs_status_string(gs_status st) {
  switch (st) {
    case GS_OK: return "ok";
    case GS_ERR_INVALID_ARG: return "invalid argument";
    case GS_ERR_OUT_OF_MEMORY: return "out of device memory";
    case GS_ERR_DEVICE: return "device error";
    case GS_ERR_UNSUPPORTED: return "unsupported";
  }
  return "unknown status";
}

const char* gs_last_error(const gs_ctx* x) { return x ? x->last_error.c_str() : g_free_error; }

gs_status gs_create(const gs_config* cfg, gs_ctx** out) {
  gs::set_free_error("");
  auto bad = [](const char* m) {
    gs::set_free_error(m);
    return GS_ERR_INVALID_ARG;
  };
  if (!out) return bad("out is NULL");
  *out = nullptr;
  if (!cfg) return bad("cfg is NULL");
  if (cfg->d < 1 || cfg->d > kP - 1) return bad("d must satisfy 1 <= d <= 2^31 - 2");
  if (cfg->P < 1 || cfg->P > GS_MAX_WORKERS) return bad("P must satisfy 1 <= P <= GS_MAX_WORKERS");
  if (cfg->r < 1 || cfg->r > GS_MAX_ROWS) return bad("r must satisfy 1 <= r <= GS_MAX_ROWS");
  if (cfg->c < 1 || cfg->c > kP - 1) return bad("c must satisfy 1 <= c <= 2^31 - 2");
  if (cfg->k_max < 1 || cfg->k_max > cfg->d) return bad("k_max must satisfy 1 <= k_max <= d");
  if (!std::isfinite(cfg->rho)) return bad("rho must be finite");
  if (!cfg->hash_a || !cfg->hash_b || !cfg->sign_a || !cfg->sign_b) return bad("hash parameter array is NULL");
  if (!valid_ab(cfg->hash_a, cfg->hash_b, cfg->r) || !valid_ab(cfg->sign_a, cfg->sign_b, cfg->r))
    return bad("hash parameters must satisfy 1 <= a < p and 0 <= b < p");
  if ((int64_t)cfg->P * cfg->r * cfg->c > (int64_t)1 << 40) return bad("P*r*c too large");
  if (cfg->state_layout != GS_STATE_WORKER_MAJOR && cfg->state_layout != GS_STATE_INTERLEAVED)
    return bad("state_layout must be GS_STATE_WORKER_MAJOR or GS_STATE_INTERLEAVED");
  if (cfg->options & ~GS_OPT_ROW_COPY) return bad("options: unknown bits");

  gs_ctx* x = new (std::nothrow) gs_ctx();
  if (!x) {
    gs::set_free_error("host allocation failed");
    return GS_ERR_OUT_OF_MEMORY;
  }
  x->d = cfg->d;
  x->c = cfg->c;
  x->k_max = cfg->k_max;
  x->P = cfg->P;
  x->r = cfg->r;
  x->rho = cfg->rho;
  x->reset_momentum = cfg->reset_momentum ? 1 : 0;
  x->state_layout = cfg->state_layout;
  x->state_stride = GS_STATE_STRIDE(cfg->P);
  x->hs.r = cfg->r;
  for (int j = 0; j < cfg->r; ++j) {
    x->hs.row[j].a = cfg->hash_a[j];
    x->hs.row[j].b = cfg->hash_b[j];
    x->hs.row[j].a2 = cfg->sign_a[j];
    x->hs.row[j].b2 = cfg->sign_b[j];
  }
  gs::set_divisor(x->hs, (uint32_t)cfg->c);

  hipError_t e = hipGetDevice(&x->device);
  if (e == hipSuccess) {
    hipDeviceProp_t prop;
    e = hipGetDeviceProperties(&prop, x->device);
    if (e == hipSuccess) x->num_cus = prop.multiProcessorCount > 0 ? prop.multiProcessorCount : 256;
  }
  if (e != hipSuccess) {
    gs::set_free_error((std::string("HIP device query failed: ") + hipGetErrorString(e)).c_str());
    delete x;
    return GS_ERR_DEVICE;
  }

  x->cand_cap = x->d;
  x->emit_blocks = gs::emit_blocks_for(x->d);
  const int64_t words = (x->d + 31) / 32;
  hipError_t ea = hipSuccess;
  auto chk = [&](hipError_t r) {
    if (ea == hipSuccess) ea = r;
  };
  chk(alloc(&x->keys, x->d));
  chk(alloc(&x->hist, gs::kDigit1Bins));
  chk(alloc(&x->hist2, gs::kDigitBins));
  chk(alloc(&x->hist_s, gs::kDigit1Bins));
  chk(alloc(&x->hist_c, gs::kDigit1Bins));
  chk(alloc(&x->ctl, 1));
  chk(alloc(&x->stage_idx, x->d));
  chk(alloc(&x->cand_key, x->cand_cap));
  chk(alloc(&x->cand_idx, x->cand_cap));
  chk(alloc(&x->bitmap, words));
  chk(alloc(&x->emit_flags, x->emit_blocks));
  chk(alloc(&x->sample_keys, gs::kSampleMax));
  x->heavy_row = (x->c + 63) / 64 * 64;
  chk(alloc(&x->heavy, (int64_t)x->r * x->heavy_row / 32));
  {
    const int64_t npad = gs::l2_pad(x->c);
    x->l2_half = (int64_t)x->r * (npad > 2048 ? npad / 2048 : 1);
    chk(alloc(&x->l2buf, 2 * x->l2_half));
  }
  x->plan = gs::make_pull_plan(x->hs, x->d, x->P, x->r, x->c, x->num_cus);
  x->use_pull = (int64_t)x->plan.T * (int64_t)sizeof(uint32_t) <= gs::kMaxFillLds;
  {
    // diagnostic overrides: GS_SKETCH_PATH=atomic selects the fp64-atomic sketch for any plan,
    // GS_SKETCH_PATH=unpacked keeps the gather's lists unpacked (coordinates and codes)
    const char* path = std::getenv("GS_SKETCH_PATH");
    if (path && std::strcmp(path, "atomic") == 0) x->use_pull = false;
    if (path && std::strcmp(path, "unpacked") == 0) x->plan.off_bits = 0;
    // GS_SELECT_PATH=pruned prunes every selection without an estimate vector, =full none
    x->prune_min_cells = gs::kPruneMinCells;
    const char* sel = std::getenv("GS_SELECT_PATH");
    if (sel && std::strcmp(sel, "pruned") == 0) x->prune_min_cells = 0;
    if (sel && std::strcmp(sel, "full") == 0) x->prune_min_cells = INT64_MAX;
    // GS_EMIT_SPIN=n bounds the emit's look-back polls (0: count directly as soon as a
    // predecessor has not published; negative: always count directly), for tests
    const char* spin = std::getenv("GS_EMIT_SPIN");
    if (spin) x->emit_spin = std::atoi(spin);
  }
  if (x->use_pull) {
    x->list_cap = (int64_t)x->r * x->d + (int64_t)gs::kListGroup * x->plan.T;
    chk(alloc(&x->list, x->list_cap));
    chk(alloc(&x->codes, x->list_cap));
    chk(alloc(&x->bases, x->list_cap / gs::kListGroup));
    chk(alloc(&x->tile_off, (int64_t)x->plan.T + 1));
    chk(alloc(&x->tile_n, (int64_t)x->plan.T));
    // the interleaved copy: the worker-major state's sketch gathers from it (with more than
    // one worker: one worker's state is a plain vector the pull gathers directly); an
    // interleaved context gathers the caller's v and needs the copy only on request
    if ((x->state_layout == GS_STATE_WORKER_MAJOR && x->P > 1) || (cfg->options & GS_OPT_ROW_COPY))
      chk(alloc(&x->vI, x->d * x->plan.PP));
    chk(alloc(&x->partial, (int64_t)x->plan.S * x->r * x->c * x->P));
  } else {
    chk(alloc(&x->acc64, (int64_t)x->P * x->r * x->c));
  }
  if (ea == hipSuccess) ea = hipMemset(x->hist, 0, gs::kDigit1Bins * sizeof(uint32_t));
  if (ea == hipSuccess) ea = hipMemset(x->hist2, 0, gs::kDigitBins * sizeof(uint32_t));
  if (ea == hipSuccess) ea = hipMemset(x->hist_s, 0, gs::kDigit1Bins * sizeof(uint32_t));
  if (ea == hipSuccess) ea = hipMemset(x->hist_c, 0, gs::kDigit1Bins * sizeof(uint32_t));
  if (ea == hipSuccess) ea = hipMemset(x->ctl, 0, sizeof(gs::SelectCtl));
  if (ea == hipSuccess) ea = hipDeviceSynchronize();
  if (ea == hipSuccess && x->use_pull) ea = gs::build_pull_lists(x);
  if (ea == hipSuccess) ea = gs::prepare_prune(x);
  if (ea != hipSuccess) {
    const bool oom = ea == hipErrorOutOfMemory || ea == hipErrorMemoryAllocation;
    gs::set_free_error((std::string("device scratch allocation failed: ") + hipGetErrorString(ea)).c_str());
    (void)hipGetLastError();
    free_scratch(x);
    delete x;
    return oom ? GS_ERR_OUT_OF_MEMORY : GS_ERR_DEVICE;
  }
  *out = x;
  return GS_OK;
}

gs_status gs_describe(const gs_ctx* x, gs_plan* out) {
  if (!x || !out) return GS_ERR_INVALID_ARG;
  gs_plan p{};
  p.sketch = x->use_pull ? GS_SKETCH_GATHER : GS_SKETCH_ATOMIC;
  p.tile_width = x->use_pull ? x->plan.W : 0;
  p.tiles = x->use_pull ? x->plan.T : 0;
  p.segments = x->use_pull ? x->plan.S : 0;
  p.packed_lists = x->use_pull ? x->plan.packed : 0;
  p.prune = x->d * x->r > x->prune_min_cells ? 1 : 0;
  p.row_copy = x->vI != nullptr ? 1 : 0;
  *out = p;
  return GS_OK;
}

gs_status gs_destroy(gs_ctx* x) {
  if (!x) return GS_OK;
  hipError_t e = hipDeviceSynchronize();
  if (x->t_events) {
    for (int64_t t = 0; t < (int64_t)x->t_max * gs::kStageMarks; ++t) (void)hipEventDestroy(x->t_events[t]);
    delete[] x->t_events;
    x->t_events = nullptr;
  }
  free_scratch(x);
  delete x;
  return e == hipSuccess ? GS_OK : GS_ERR_DEVICE;
}

gs_status gs_accumulate(gs_ctx* x, void* stream, const float* g, float* u, float* v) {
  if (!x) return GS_ERR_INVALID_ARG;
  x->last_error.clear();
  if (!g || !u || !v) return fail(x, GS_ERR_INVALID_ARG, "gs_accumulate: NULL array");
  return device_status(x, gs::launch_accumulate(x, as_stream(stream), g, u, v), "gs_accumulate");
}

gs_status gs_sketch(gs_ctx* x, void* stream, const float* v, float* tables) {
  if (!x) return GS_ERR_INVALID_ARG;
  x->last_error.clear();
  if (!v || !tables) return fail(x, GS_ERR_INVALID_ARG, "gs_sketch: NULL array");
  if (unaligned_without_copy(x, v)) return fail(x, GS_ERR_INVALID_ARG, std::string("gs_sketch") + kUnalignedMsg);
  hipStream_t s = as_stream(stream);
  hipError_t e;
  if (x->use_pull && gs::flat_state(x)) {
    e = gs::launch_pull_flat(x, s, v, nullptr, tables);
    if (e == hipSuccess) e = gs::launch_merge_partials(x, s, nullptr, tables);
  } else if (x->use_pull) {
    const float* rows = x->vI;
    if (x->state_layout == GS_STATE_INTERLEAVED)
      rows = gs::pull_rows_of_state(x, s, v, &e);
    else
      e = gs::launch_interleave(x, s, v);
    if (e == hipSuccess) e = gs::launch_pull(x, s, rows, nullptr, tables);
    if (e == hipSuccess) e = gs::launch_merge_partials(x, s, nullptr, tables);
  } else {
    e = gs::launch_sketch(x, s, v, gs::state_view(x), tables);
  }
  return device_status(x, e, "gs_sketch");
}

gs_status gs_merge(gs_ctx* x, void* stream, const float* tables, float* merged) {
  if (!x) return GS_ERR_INVALID_ARG;
  x->last_error.clear();
  if (!tables || !merged) return fail(x, GS_ERR_INVALID_ARG, "gs_merge: NULL array");
  return device_status(x, gs::launch_merge(x, as_stream(stream), tables, merged), "gs_merge");
}

gs_status gs_unsketch_topk(gs_ctx* x, void* stream, const float* merged, int64_t k, float* est, int32_t* idx) {
  if (!x) return GS_ERR_INVALID_ARG;
  x->last_error.clear();
  if (!merged || !idx) return fail(x, GS_ERR_INVALID_ARG, "gs_unsketch_topk: NULL array");
  if (k < 1 || k > x->k_max) return fail(x, GS_ERR_INVALID_ARG, "gs_unsketch_topk: k must satisfy 1 <= k <= k_max");
  return device_status(x, gs::launch_unsketch_topk(x, as_stream(stream), merged, k, est, idx), "gs_unsketch_topk");
}

gs_status gs_gather_reset(gs_ctx* x, void* stream, const int32_t* idx, int64_t k, float* u, float* v,
                          float* values) {
  if (!x) return GS_ERR_INVALID_ARG;
  x->last_error.clear();
  if (!idx || !u || !v || !values) return fail(x, GS_ERR_INVALID_ARG, "gs_gather_reset: NULL array");
  if (k < 1 || k > x->k_max) return fail(x, GS_ERR_INVALID_ARG, "gs_gather_reset: k must satisfy 1 <= k <= k_max");
  return device_status(x, gs::launch_gather_reset(x, as_stream(stream), idx, k, u, v, values), "gs_gather_reset");
}

}  // extern "C"

// accumulate + sketch + merge of the fused step (tables kept in context scratch); mark(t)
// is called before stage 0 (t = 0) and after stages 0..2 (t = 1..3)
template <class Mark>
static hipError_t launch_sketch_phase(gs_ctx* x, hipStream_t s, const float* g, float* u, float* v, float* merged,
                                      Mark mark) {
  hipError_t e;
  mark(0);
  if (x->use_pull) {
    const float* rows = x->vI;
    const bool flat = gs::flat_state(x);
    if (x->state_layout == GS_STATE_INTERLEAVED) {
      // the caller's v rows are what the pull gathers: no interleaved copy
      e = gs::launch_accumulate(x, s, g, u, v);
      if (e == hipSuccess) rows = gs::pull_rows_of_state(x, s, v, &e);
    } else if (flat) {
      e = gs::launch_accumulate(x, s, g, u, v);  // one worker: v itself is gathered
    } else {
      e = gs::launch_accumulate_vi(x, s, g, u, v);
    }
    mark(1);
    if (e == hipSuccess) e = flat ? gs::launch_pull_flat(x, s, v, merged, nullptr)
                                  : gs::launch_pull(x, s, rows, merged, nullptr);
    mark(2);
    if (e == hipSuccess) e = gs::launch_merge_partials(x, s, merged, nullptr);
  } else {
    e = gs::launch_accumulate(x, s, g, u, v);
    mark(1);
    if (e == hipSuccess) e = gs::launch_sketch_acc(x, s, v, gs::state_view(x));
    mark(2);
    if (e == hipSuccess) e = gs::launch_merge_acc(x, s, merged);
  }
  mark(3);
  return e;
}

static hipError_t launch_sketch_phase(gs_ctx* x, hipStream_t s, const float* g, float* u, float* v, float* merged) {
  return launch_sketch_phase(x, s, g, u, v, merged, [x, s](int t) { gs::stage_mark(x, s, t); });
}

extern "C" {

gs_status gs_step(gs_ctx* x, void* stream, const float* g, float* u, float* v, int64_t k, float* merged,
                  int32_t* idx, float* values) {
  if (!x) return GS_ERR_INVALID_ARG;
  x->last_error.clear();
  if (!g || !u || !v || !merged || !idx || !values) return fail(x, GS_ERR_INVALID_ARG, "gs_step: NULL array");
  if (k < 1 || k > x->k_max) return fail(x, GS_ERR_INVALID_ARG, "gs_step: k must satisfy 1 <= k <= k_max");
  if (unaligned_without_copy(x, v)) return fail(x, GS_ERR_INVALID_ARG, std::string("gs_step") + kUnalignedMsg);
  hipStream_t s = as_stream(stream);
  hipError_t e = launch_sketch_phase(x, s, g, u, v, merged);
  if (e == hipSuccess) e = gs::launch_unsketch_topk(x, s, merged, k, nullptr, idx);
  gs::stage_mark(x, s, 4);
  if (e == hipSuccess) e = gs::launch_gather_reset(x, s, idx, k, u, v, values);
  gs::stage_mark(x, s, 5);
  return device_status(x, e, "gs_step");
}

gs_status gs_heavymix_topk(gs_ctx* x, void* stream, const float* merged, int64_t k, const uint32_t* rnd, float* est,
                           int32_t* idx, int64_t* n_heavy, double* l2sq) {
  if (!x) return GS_ERR_INVALID_ARG;
  x->last_error.clear();
  if (!merged || !rnd || !idx) return fail(x, GS_ERR_INVALID_ARG, "gs_heavymix_topk: NULL array");
  if (k < 1 || k > x->k_max) return fail(x, GS_ERR_INVALID_ARG, "gs_heavymix_topk: k must satisfy 1 <= k <= k_max");
  return device_status(x, gs::launch_heavymix_topk(x, as_stream(stream), merged, k, rnd, est, idx, n_heavy, l2sq),
                       "gs_heavymix_topk");
}

gs_status gs_step_heavymix(gs_ctx* x, void* stream, const float* g, float* u, float* v, int64_t k,
                           const uint32_t* rnd, float* merged, int32_t* idx, float* values, int64_t* n_heavy) {
  if (!x) return GS_ERR_INVALID_ARG;
  x->last_error.clear();
  if (!g || !u || !v || !rnd || !merged || !idx || !values)
    return fail(x, GS_ERR_INVALID_ARG, "gs_step_heavymix: NULL array");
  if (k < 1 || k > x->k_max) return fail(x, GS_ERR_INVALID_ARG, "gs_step_heavymix: k must satisfy 1 <= k <= k_max");
  if (unaligned_without_copy(x, v))
    return fail(x, GS_ERR_INVALID_ARG, std::string("gs_step_heavymix") + kUnalignedMsg);
  hipStream_t s = as_stream(stream);
  hipError_t e = launch_sketch_phase(x, s, g, u, v, merged);
  if (e == hipSuccess) e = gs::launch_heavymix_topk(x, s, merged, k, rnd, nullptr, idx, n_heavy, nullptr);
  gs::stage_mark(x, s, 4);
  if (e == hipSuccess) e = gs::launch_gather_reset(x, s, idx, k, u, v, values);
  gs::stage_mark(x, s, 5);
  return device_status(x, e, "gs_step_heavymix");
}

gs_status gs_step_sketch_momentum(gs_ctx* x, void* stream, const float* g, float* U, float* E, int64_t k,
                                  float* merged, int32_t* idx, float* values) {
  if (!x) return GS_ERR_INVALID_ARG;
  x->last_error.clear();
  if (!g || !U || !E || !merged || !idx || !values)
    return fail(x, GS_ERR_INVALID_ARG, "gs_step_sketch_momentum: NULL array");
  if (k < 1 || k > x->k_max)
    return fail(x, GS_ERR_INVALID_ARG, "gs_step_sketch_momentum: k must satisfy 1 <= k <= k_max");
  if (x->use_pull && x->P > 1 && x->vI == nullptr)
    return fail(x, GS_ERR_UNSUPPORTED,
                "gs_step_sketch_momentum: an interleaved-state context needs the row copy (GS_OPT_ROW_COPY)");
  hipStream_t s = as_stream(stream);
  hipError_t e;
  gs::stage_mark(x, s, 0);
  if (x->use_pull && x->P == 1) {  // one worker's gradient [1][d] is a plain vector: gathered directly
    gs::stage_mark(x, s, 1);
    e = gs::launch_pull_flat(x, s, g, merged, nullptr);
    gs::stage_mark(x, s, 2);
    if (e == hipSuccess) e = gs::launch_merge_partials(x, s, merged, nullptr);
  } else if (x->use_pull) {
    e = gs::launch_interleave(x, s, g);
    gs::stage_mark(x, s, 1);
    if (e == hipSuccess) e = gs::launch_pull(x, s, x->vI, merged, nullptr);
    gs::stage_mark(x, s, 2);
    if (e == hipSuccess) e = gs::launch_merge_partials(x, s, merged, nullptr);
  } else {
    gs::stage_mark(x, s, 1);
    e = gs::launch_sketch_acc(x, s, g, gs::worker_major_view(x));
    gs::stage_mark(x, s, 2);
    if (e == hipSuccess) e = gs::launch_merge_acc(x, s, merged);
  }
  gs::stage_mark(x, s, 3);
  if (e == hipSuccess) e = gs::launch_sketch_state(x, s, merged, U, E, k, idx, values);  // marks 4 and 5
  return device_status(x, e, "gs_step_sketch_momentum");
}

gs_status gs_apply_update(gs_ctx* x, void* stream, const int32_t* idx, const float* values, int64_t k, float lr,
                          float* w) {
  if (!x) return GS_ERR_INVALID_ARG;
  x->last_error.clear();
  if (!idx || !values || !w) return fail(x, GS_ERR_INVALID_ARG, "gs_apply_update: NULL array");
  if (k < 1 || k > x->k_max) return fail(x, GS_ERR_INVALID_ARG, "gs_apply_update: k must satisfy 1 <= k <= k_max");
  if (!std::isfinite(lr)) return fail(x, GS_ERR_INVALID_ARG, "gs_apply_update: lr must be finite");
  return device_status(x, gs::launch_apply_update(x, as_stream(stream), idx, values, k, lr, w), "gs_apply_update");
}

gs_status gs_timing_start(gs_ctx* x, int32_t max_steps) {
  if (!x) return GS_ERR_INVALID_ARG;
  x->last_error.clear();
  if (x->timing) return fail(x, GS_ERR_INVALID_ARG, "gs_timing_start: timing already active");
  if (max_steps < 1 || max_steps > (1 << 20)) return fail(x, GS_ERR_INVALID_ARG, "gs_timing_start: bad max_steps");
  const int64_t n = (int64_t)max_steps * gs::kStageMarks;
  hipEvent_t* ev = new (std::nothrow) hipEvent_t[n]();
  if (!ev) return fail(x, GS_ERR_OUT_OF_MEMORY, "gs_timing_start: host allocation failed");
  hipError_t e = hipSuccess;
  int64_t made = 0;
  for (; made < n && e == hipSuccess; ++made) e = hipEventCreate(&ev[made]);
  if (e != hipSuccess) {
    for (int64_t t = 0; t < made; ++t)
      if (ev[t]) (void)hipEventDestroy(ev[t]);
    delete[] ev;
    return device_status(x, e, "gs_timing_start");
  }
  x->t_events = ev;
  x->t_max = max_steps;
  x->t_step = 0;
  x->timing = true;
  return GS_OK;
}

gs_status gs_timing_stop(gs_ctx* x, float* stage_ms, int32_t* n_steps) {
  if (!x) return GS_ERR_INVALID_ARG;
  x->last_error.clear();
  if (!x->timing) return fail(x, GS_ERR_INVALID_ARG, "gs_timing_stop: timing not active");
  const int32_t steps = x->t_step;
  hipError_t e = hipSuccess;
  double acc[GS_NUM_STAGES] = {0.0, 0.0, 0.0, 0.0, 0.0};
  for (int32_t st = 0; st < steps && e == hipSuccess; ++st) {
    hipEvent_t* m = x->t_events + (int64_t)st * gs::kStageMarks;
    e = hipEventSynchronize(m[gs::kStageMarks - 1]);
    for (int t = 0; t < GS_NUM_STAGES && e == hipSuccess; ++t) {
      float ms = 0.f;
      e = hipEventElapsedTime(&ms, m[t], m[t + 1]);
      acc[t] += ms;
    }
  }
  for (int64_t t = 0; t < (int64_t)x->t_max * gs::kStageMarks; ++t) (void)hipEventDestroy(x->t_events[t]);
  delete[] x->t_events;
  x->t_events = nullptr;
  x->timing = false;
  x->t_max = x->t_step = 0;
  if (e != hipSuccess) return device_status(x, e, "gs_timing_stop");
  if (stage_ms)
    for (int t = 0; t < GS_NUM_STAGES; ++t) stage_ms[t] = steps ? (float)(acc[t] / steps) : 0.f;
  if (n_steps) *n_steps = steps;
  return GS_OK;
}

gs_status gs_step_profiled(gs_ctx* x, void* stream, const float* g, float* u, float* v, int64_t k, float* merged,
                           int32_t* idx, float* values, float* stage_ms) {
  if (!x) return GS_ERR_INVALID_ARG;
  x->last_error.clear();
  if (!g || !u || !v || !merged || !idx || !values || !stage_ms)
    return fail(x, GS_ERR_INVALID_ARG, "gs_step_profiled: NULL array");
  if (k < 1 || k > x->k_max) return fail(x, GS_ERR_INVALID_ARG, "gs_step_profiled: k must satisfy 1 <= k <= k_max");
  if (unaligned_without_copy(x, v))
    return fail(x, GS_ERR_INVALID_ARG, std::string("gs_step_profiled") + kUnalignedMsg);
  hipStream_t s = as_stream(stream);
  hipEvent_t ev[GS_NUM_STAGES + 1] = {};
  hipError_t e = hipSuccess;
  for (int t = 0; t <= GS_NUM_STAGES && e == hipSuccess; ++t) e = hipEventCreate(&ev[t]);
  hipError_t erec = hipSuccess;
  auto mark = [&](int t) {
    if (erec == hipSuccess) erec = hipEventRecord(ev[t], s);
  };
  if (e == hipSuccess) e = launch_sketch_phase(x, s, g, u, v, merged, mark);
  if (e == hipSuccess) e = gs::launch_unsketch_topk(x, s, merged, k, nullptr, idx);
  mark(4);
  if (e == hipSuccess) e = gs::launch_gather_reset(x, s, idx, k, u, v, values);
  mark(5);
  if (e == hipSuccess) e = erec;
  if (e == hipSuccess) e = hipEventSynchronize(ev[5]);
  for (int t = 0; t < GS_NUM_STAGES && e == hipSuccess; ++t) e = hipEventElapsedTime(&stage_ms[t], ev[t], ev[t + 1]);
  for (int t = 0; t <= GS_NUM_STAGES; ++t)
    if (ev[t]) (void)hipEventDestroy(ev[t]);
  return device_status(x, e, "gs_step_profiled");
}

}  // extern "C"
