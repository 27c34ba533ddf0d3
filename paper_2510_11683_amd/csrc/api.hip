// Host orchestration and the C ABI of libbgpo.
//
// One call walks the Monte-Carlo samples j of its range in order (Algorithm 1,
// inner loop), in units of up to G consecutive samples: draw t and the mask of
// each sample of the unit, compact its masked rows after those of the unit's
// earlier samples and gather them (through the final RMSNorm for the _rmsnorm
// calls), run the fused LM-head forward once over the unit's rows (with
// backward it also keeps the exponentials of the logits), form l, d, g and
// the gradient scale of every (sample, response), turn the exponentials into
// dZ = s (softmax - onehot), run one dX GEMM over the unit's rows and add each
// sample's rows into dX in sample order; dW is accumulated once per batch of
// units.  Under a small workspace budget the backward instead recomputes the
// logits one vocabulary chunk at a time (nothing of size rows x V is kept) and
// accumulates dX and dW chunk by chunk.  The
// samples stay independent (the bound is a sum over samples, Eq.
// lower_bound_def): a unit only shares the GEMM launches, which saves the
// padded rows and partly filled GEMM rounds of one sample at a time.  All
// buffers are views into the caller's workspace, sized by B, L, d, V, the
// input type and the budget; nothing depends on n_t, so device memory is the
// same for any number of
// samples (except in the retained-state contrast mode of the exact
// objective).
#include <math.h>
#include <string.h>

#include <algorithm>
#include <mutex>
#include <vector>

#include "../../include/bgpo.h"
#include "internal.hpp"

namespace bgpo {

static size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

constexpr int64_t kMaxUnit = 8;
constexpr int64_t kDwUnits = 2;   // units per dW GEMM in the constant-memory mode
// units per dW GEMM that a workspace budget above the default layout may buy
// (each halving of the dW read-modify-writes saves about 1 % of the step at
// the LLaDA head shape)
constexpr int64_t kDwUnitsMax = 4;
constexpr int64_t kGiB = int64_t(1) << 30;

static int64_t padded_positions(const Dims& dm) {
  const int64_t P = (int64_t)dm.B * dm.L;
  return (P + kRowPad - 1) / kRowPad * kRowPad;
}

// largest unit whose row capacity stays within the row kernels' grid (65535
// workgroups of 64 rows)
static int64_t max_unit(const Dims& dm) {
  return std::max<int64_t>(1, std::min<int64_t>(kMaxUnit, int64_t(65535) * 64 / padded_positions(dm)));
}

size_t workspace_layout(const Dims& dm, const Plan& pl, void* base, Workspace* ws,
                        Workspace* units) {
  const int64_t P = (int64_t)dm.B * dm.L;
  const int64_t NP = padded_positions(dm);
  const int64_t nvt = (dm.V + kVocabTile - 1) / kVocabTile;
  const int64_t G = pl.G;
  const int64_t n_units = pl.retain ? (dm.n_t + G - 1) / G : 1;
  const int64_t RP = G * NP;
  const int64_t dw_batch = pl.retain ? n_units : pl.dw_batch;
  // the rows of a dW batch: columns of H_c^T, rows of the stored dZ
  const int64_t KT = dw_batch * RP;
  const int64_t chunk = pl.chunk;

  size_t off = 0;
  char* b = static_cast<char*>(base);
  auto take = [&](size_t bytes) -> void* {
    void* p = b ? b + off : nullptr;
    off = align_up(off + bytes, 256);
    return p;
  };
  // the state of one unit: masks and rows, log-sum-exp partials, H_c (and a
  // vocabulary chunk's dZ).  Every unit's state comes first, at the head of
  // the workspace: the forward GEMM reads H_c one K slab (rows x 128 bytes)
  // after another, a new span of memory per slab, and with H_c at the tail
  // of a large allocation the forward ran up to 5 % slower (measured), at
  // its head not.
  auto take_unit = [&](Workspace& w) {
    w.meta = static_cast<SampleMeta*>(take(G * sizeof(SampleMeta)));
    w.idx = static_cast<int32_t*>(take(G * P * 4));
    w.row_tgt = static_cast<int32_t*>(take(RP * 4));
    w.row_seq = static_cast<int32_t*>(take(RP * 4));
    w.seg_off = static_cast<int32_t*>(take(G * (dm.B + 1) * 4));
    w.t24 = static_cast<uint32_t*>(take(G * dm.B * 4));
    w.seq_scale = static_cast<float*>(take(G * dm.B * 4));
    w.ztgt = static_cast<float*>(take(RP * 4));
    w.lse2 = static_cast<float*>(take(RP * 4));
    w.lp = static_cast<float*>(take(RP * 4));
    w.row_scale = static_cast<float*>(take(RP * 4));
    w.row_f = static_cast<float*>(take(RP * 4));
    w.row_bad = static_cast<uint8_t*>(take(RP));
    w.inv_rms = static_cast<float*>(take(RP * 4));
    w.mask_scratch = take(mask_scratch_bytes(dm.B, dm.L));
    w.part_m = static_cast<float*>(take(nvt * RP * 4));
    w.part_s = static_cast<float*>(take(nvt * RP * 4));
    w.Hc = static_cast<uint16_t*>(take(RP * dm.d * 2));
    if (chunk) w.dZ = static_cast<uint16_t*>(take(RP * chunk * 2));
  };
  Workspace w{};
  take_unit(w);
  const size_t unit_bytes = off;   // the same for every unit (all pieces 256-byte aligned)
  off = unit_bytes * n_units;
  w.dbar = static_cast<double*>(take(dm.B * 8));
  w.gpart = static_cast<float*>(take((NP / 256) * dm.d * 4));
  w.HcT = static_cast<uint16_t*>(take(KT * dm.d * 2));
  w.WT = static_cast<uint16_t*>(take((size_t)dm.V * dm.d * 2));
  // the slab-major bf16 W of the dX GEMM (without it the GEMM reads the
  // caller's bf16 W in place)
  w.Wk = pl.w_copy ? static_cast<uint16_t*>(take((size_t)dm.V * dm.d * 2)) : nullptr;
  w.ldz = chunk ? RP : KT + kDzPadRows;
  if (!chunk) w.dZ = static_cast<uint16_t*>(take(w.ldz * dm.V * 2));
  w.dx_part = static_cast<float*>(take(pl.n_split * RP * dm.d * 4));
  w.P = P;
  w.NP = NP;
  w.nvt = nvt;
  w.G = G;
  w.RP = RP;
  w.n_split = pl.n_split;
  w.dw_batch = dw_batch;
  w.KT = KT;
  w.chunk = chunk;
  w.g_used = (int)G;
  const size_t end = off;
  for (int64_t u = 1; u < n_units; ++u) {
    Workspace wu = w;
    off = unit_bytes * u;
    take_unit(wu);
    if (units) units[u] = wu;
  }
  off = end;
  if (units) units[0] = w;
  if (ws) *ws = w;
  return off;
}

static size_t plan_bytes(const Dims& dm, const Plan& pl) {
  return workspace_layout(dm, pl, nullptr, nullptr, nullptr);
}

// The stored-exponential plan used without a budget: units of up to 8
// samples while the unit's H_c and the dZ rows and H_c^T columns of a dW
// batch of two units stay within about 32 GB; dX split capacity up to 16
// within about 4 GB.  With every sample retained, the same units (at most n_t
// samples each) each keep their own state and all of them form the one dW
// batch, so both modes run the same unit compositions.
static Plan default_plan(const Dims& dm, int retain) {
  const int64_t NP = padded_positions(dm);
  const int64_t per_sample = NP * ((int64_t)dm.V * kDwUnits + (int64_t)dm.d * (1 + kDwUnits)) * 2;
  int64_t G = std::max<int64_t>(1, std::min(max_unit(dm), 32 * kGiB / per_sample));
  if (retain) G = std::min<int64_t>(G, dm.n_t);
  const int64_t RP = G * NP;
  const int64_t n_split = std::max<int64_t>(1, std::min<int64_t>(16, 4 * kGiB / (RP * dm.d * 4)));
  const int64_t dw_batch = kDwUnits * RP <= kMaxColumns ? kDwUnits : 1;
  return Plan{G, dw_batch, n_split, 0, retain, 1};
}

// Estimated time (arbitrary units) per sample of the recompute backward for
// a plan: the four GEMM passes at the fill of a 256-workgroup grid (tiles for
// about half of the positions masked, as E[t] = 1/2), plus the fp32
// read-modify-write traffic that the chunking adds (dX partials once per
// chunk and split, dW once per unit).  Used only to rank plans.
// The grid fill of a GEMM of `tiles` tiles on 256 workgroups, averaged over
// masked fractions 0.4 .. 0.6 of the positions (rows_t row tiles at 0.5)
static double mean_fill(double rows_cap, double other_tiles, double split) {
  double f = 0.0;
  for (double q : {0.4, 0.45, 0.5, 0.55, 0.6}) {
    const double tiles = std::max(1.0, std::ceil(rows_cap * q / 256.0)) * other_tiles * split;
    f += tiles / (256.0 * std::ceil(tiles / 256.0));
  }
  return f / 5.0;
}

static double recompute_cost(const Dims& dm, const Plan& pl) {
  const double NP = (double)padded_positions(dm);
  const double rows = pl.G * NP;
  const double col_t = std::ceil(dm.d / 256.0);
  const double chunk_t = std::ceil(pl.chunk / 256.0);
  const double n_chunks = std::ceil((double)dm.V / pl.chunk);
  const double pass = 2.0 * NP * 0.5 * dm.d * (double)dm.V / 1.35e15;   // s per sample per pass
  // forward (whole vocabulary: well filled), recompute, dX, dW (its tiles
  // span the chunk and d, not the rows)
  const double dw_tiles = chunk_t * col_t;
  const double dw_fill = dw_tiles / (256.0 * std::ceil(dw_tiles / 256.0));
  const double gemm = pass * (1.0 + 1.0 / mean_fill(rows, chunk_t, 1.0) +
                              1.0 / mean_fill(rows, col_t, (double)pl.n_split) + 1.0 / dw_fill);
  const double rmw = (n_chunks * NP * 0.5 * dm.d * 8.0 * pl.n_split + (double)dm.V * dm.d * 8.0 / pl.G) /
                     5e12;
  return gemm + rmw;
}

// The same estimate for the stored-exponential backward: three GEMM passes
// (the dX GEMM at the best split the capacity allows, about 2 % faster on
// the slab-major copy of W), the forward's stores of the kept exponentials
// (2 bytes per entry) and the dW read-modify-write once per batch of units.
static double stored_cost(const Dims& dm, const Plan& pl) {
  const double NP = (double)padded_positions(dm);
  const double rows = pl.G * NP;
  const double col_t = std::ceil(dm.d / 256.0);
  double dx_fill = 0.0;
  for (int64_t sp = 1; sp <= pl.n_split; ++sp)
    dx_fill = std::max(dx_fill, mean_fill(rows, col_t, (double)sp));
  const double pass = 2.0 * NP * 0.5 * dm.d * (double)dm.V / 1.35e15;
  const double dx_rate = pl.w_copy ? 0.98 : 1.0;
  const double gemm =
      pass * (1.0 / mean_fill(rows, std::ceil(dm.V / 256.0), 1.0) + dx_rate / dx_fill + 1.0);
  const double mem = (2.0 * NP * 0.5 * dm.V + (double)dm.V * dm.d * 8.0 / (pl.G * pl.dw_batch)) / 5e12;
  return gemm + mem;
}

// Chooses the plan of a problem (see bgpo.h: backward modes and the workspace
// budget).  Returns BGPO_OK, or BGPO_ERR_BUDGET when nothing fits the budget.
static int choose_plan(const bgpo_problem* p, Plan* out) {
  const Dims dm{p->B, p->L, p->d, p->V, p->n_t};
  const int f32 = p->in_dtype == BGPO_F32;
  const uint64_t budget = p->ws_budget;
  if (p->retain_samples || (budget == 0 && p->vocab_chunk == 0)) {
    *out = default_plan(dm, p->retain_samples);
    return BGPO_OK;
  }
  const int64_t NP = padded_positions(dm);
  if (p->vocab_chunk == 0) {
    // the default layout if it fits (with the largest dW batch the budget
    // allows on top of it), else the stored-mode layout of least estimated
    // time that fits
    const Plan dflt = default_plan(dm, 0);
    if (plan_bytes(dm, dflt) <= budget) {
      *out = dflt;
      for (int64_t dwb = kDwUnitsMax; dwb > dflt.dw_batch; --dwb) {
        Plan pl = dflt;
        pl.dw_batch = dwb;
        if (dwb * dflt.G * NP <= kMaxColumns && plan_bytes(dm, pl) <= budget) {
          *out = pl;
          break;
        }
      }
      return BGPO_OK;
    }
    bool found = false;
    Plan best{};
    double best_cost = 0.0;
    for (int64_t G = max_unit(dm); G >= 1; --G) {
      for (int64_t dwb = kDwUnits; dwb >= 1; --dwb) {
        if (dwb * G * NP > kMaxColumns) continue;
        const int64_t ns_max = std::max<int64_t>(1, std::min<int64_t>(16, 4 * kGiB / (G * NP * p->d * 4)));
        for (int wc = 1; wc >= f32; --wc) {   // with and (bf16 inputs) without the W copy
          for (int64_t ns = 1; ns <= ns_max; ++ns) {
            const Plan pl{G, dwb, ns, 0, 0, wc};
            if (plan_bytes(dm, pl) > budget) break;   // more splits only take more memory
            const double c = stored_cost(dm, pl);
            if (!found || c < best_cost) {
              found = true;
              best = pl;
              best_cost = c;
            }
          }
        }
      }
    }
    if (found) {
      *out = best;
      return BGPO_OK;
    }
  }
  // recompute mode: the cheapest (unit, chunk, split capacity) that fits the
  // budget (or about 32 GB without one)
  const uint64_t cap = budget ? budget : (uint64_t)(32 * kGiB);
  const int64_t v_round = ((int64_t)p->V + 255) / 256 * 256;
  std::vector<int64_t> widths;
  if (p->vocab_chunk) {
    widths.push_back(std::min<int64_t>(p->vocab_chunk, v_round));
  } else {
    for (int64_t c : {32768, 16384, 8192, 4096, 2048, 1024, 512, 256}) {
      const int64_t w = std::min<int64_t>(c, v_round);
      if (widths.empty() || widths.back() != w) widths.push_back(w);
    }
  }
  bool found = false;
  Plan best{};
  double best_cost = 0.0;
  for (int64_t G = max_unit(dm); G >= 1; --G) {
    if (G * NP > kMaxColumns) continue;
    for (int64_t C : widths) {
      for (int64_t ns : {4, 2, 1}) {
        const Plan pl{G, 1, ns, C, 0, f32};
        if (plan_bytes(dm, pl) > cap) continue;
        const double c = recompute_cost(dm, pl);
        if (!found || c < best_cost) {
          found = true;
          best = pl;
          best_cost = c;
        }
      }
    }
  }
  if (!found) return BGPO_ERR_BUDGET;
  *out = best;
  return BGPO_OK;
}

// HIP-event timing of kernel classes, enabled by a non-NULL record.
class Timer {
 public:
  Timer(bgpo_timing* out, hipStream_t s) : out_(out), s_(s) {}
  ~Timer() {
    // best-effort release; a failure here cannot be reported from a destructor
    for (auto& e : ev_) {
      if (e.a) (void)hipEventDestroy(e.a);
      if (e.b) (void)hipEventDestroy(e.b);
    }
  }
  hipError_t begin(int kind) {
    if (!out_) return hipSuccess;
    Ev e{kind, 0, nullptr, nullptr};
    hipError_t r = hipEventCreate(&e.a);
    if (r == hipSuccess) r = hipEventCreate(&e.b);
    if (r == hipSuccess) r = hipEventRecord(e.a, s_);
    ev_.push_back(e);
    return r;
  }
  // closes the range opened by the last begin(); `launches` kernels ran in it
  hipError_t end(int launches = 1) {
    if (!out_) return hipSuccess;
    ev_.back().launches = launches;
    return hipEventRecord(ev_.back().b, s_);
  }
  hipError_t finish() {
    if (!out_ || ev_.empty()) return hipSuccess;
    hipError_t r = hipEventSynchronize(ev_.back().b);
    if (r != hipSuccess) return r;
    for (auto& e : ev_) {
      float ms = 0.f;
      r = hipEventElapsedTime(&ms, e.a, e.b);
      if (r != hipSuccess) return r;
      out_->ms[e.kind] += ms;
      out_->launches[e.kind] += e.launches;
    }
    return hipSuccess;
  }

 private:
  struct Ev {
    int kind, launches;
    hipEvent_t a, b;
  };
  bgpo_timing* out_;
  hipStream_t s_;
  std::vector<Ev> ev_;
};

// Validates a problem and chooses its plan (the layout its workspace takes).
static int plan_problem(const bgpo_problem* p, Plan* pl) {
  if (!p) return BGPO_ERR_INVALID_ARG;
  if (p->B < 1 || p->L < 1 || p->n_t < 1 || p->j_begin < 0 || p->j_count < 0 ||
      (int64_t)p->j_begin + p->j_count > p->n_t || (p->t_mode != BGPO_T_IID && p->t_mode != BGPO_T_STRATIFIED) ||
      p->bound < BGPO_BOUND_PAPER || p->bound > BGPO_BOUND_EXACT || p->d < 1 || p->V < 1 ||
      p->sample_stride < 0 || p->sample_stride % 8 || !isfinite(p->norm_eps) || p->norm_eps < 0.f ||
      (p->retain_samples != 0 && p->retain_samples != 1) ||
      (p->retain_samples && p->bound != BGPO_BOUND_EXACT) ||
      (p->in_dtype != BGPO_BF16 && p->in_dtype != BGPO_F32) || p->vocab_chunk < 0 ||
      p->vocab_chunk % 256 || (p->retain_samples && (p->vocab_chunk || p->ws_budget)))
    return BGPO_ERR_INVALID_ARG;
  if (p->B > 4096 || (int64_t)p->B * p->L > (1 << 20) || p->d % 64 || p->V % 64 || p->d < 64 ||
      p->d > 65536 || p->V < 64 || p->V > (1 << 20))
    return BGPO_ERR_UNSUPPORTED;
  const int st = choose_plan(p, pl);
  if (st != BGPO_OK) return st;
  // H_c^T holds KT columns and the stored dZ KT rows (32-bit offsets in the
  // sample records).  One unit's row capacity stays within 65535 * 64 by
  // construction; with every sample retained KT grows with n_t and is
  // bounded here.
  static_assert(int64_t(65535) * 64 / 256 * 256 * kDwUnitsMax <= kMaxColumns,
                "constant-mode KT must fit the column range");
  Workspace w;
  workspace_layout(Dims{p->B, p->L, p->d, p->V, p->n_t}, *pl, nullptr, &w, nullptr);
  if (w.KT > kMaxColumns) return BGPO_ERR_UNSUPPORTED;
  return BGPO_OK;
}

static Dims dims_of(const bgpo_problem* p) { return Dims{p->B, p->L, p->d, p->V, p->n_t}; }

#define BGPO_TRY(expr)                       \
  do {                                       \
    if ((expr) != hipSuccess) return BGPO_ERR_HIP; \
  } while (0)

// the dX GEMM's K: the whole vocabulary, or one chunk of it in the recompute mode
static DxPlan dx_plan(const Dims& dm, const Workspace& ws, int grid) {
  const int k = ws.chunk ? (int)std::min<int64_t>(ws.chunk, dm.V) : dm.V;
  return DxPlan{k / 64, (dm.d + 255) / 256, grid, (int)ws.n_split};
}

// The head input of the samples of a call: sample j reads x + (j - j_begin) *
// stride elements (stride 0: one tensor shared by all samples; bf16 or, with
// f32, fp32 elements), normalised by the final RMSNorm when gamma is given.
struct Act {
  const void* x;
  bool f32;
  const float* gamma;
  float eps;
  int64_t stride;
  int j0;
  const void* at(int j) const {
    const int64_t off = (int64_t)(j - j0) * stride;
    return f32 ? (const void*)(static_cast<const float*>(x) + off)
               : (const void*)(static_cast<const uint16_t*>(x) + off);
  }
};

// forward part of the unit of samples j0 .. j0 + n_s - 1: masks .. l (and,
// with backward, g / loss / scale); prev_unit: record of the previous unit of
// the dW batch (NULL for the first)
static int run_forward_unit(const bgpo_problem* p, Workspace& ws, Timer& tm, int grid, int j0,
                            int n_s, const Act& act, const int32_t* targets, const uint8_t* resp,
                            const float* adv, const double* ell_old, double loss_scale,
                            double* ell, double* g, double* loss, int32_t* n_masked, float* t_out,
                            int32_t* flags, bool backward, bool store_u,
                            const SampleMeta* prev_unit, const double* dbar, hipStream_t s) {
  const Dims dm = dims_of(p);
  ws.g_used = n_s;
  BGPO_TRY(tm.begin(BGPO_K_MASK));
  for (int gs = 0; gs < n_s; ++gs) {
    const int j = j0 + gs;
    BGPO_TRY(launch_mask_compact(resp, targets, dm.B, dm.L, dm.n_t, j, gs, p->t_mode, p->seed,
                                 p->seq_id_base, &ws, nullptr, n_masked + j, dm.n_t,
                                 t_out ? t_out + j : nullptr, dm.n_t, dm.V,
                                 gs ? ws.meta + (gs - 1) : prev_unit, dx_plan(dm, ws, grid),
                                 ws.mask_scratch, false, s));
  }
  BGPO_TRY(tm.end(n_s));
  BGPO_TRY(tm.begin(BGPO_K_GATHER));
  if (act.gamma)
    BGPO_TRY(launch_row_rms(act.at(j0), act.f32, act.stride, dm.B, ws, dm.d, act.eps, s));
  BGPO_TRY(launch_gather(act.at(j0), act.f32, act.stride, dm.B, act.gamma, ws, dm.d, s));
  BGPO_TRY(tm.end(act.gamma ? 2 : 1));
  // the target logits first: the stored forward's exponent reference
  BGPO_TRY(tm.begin(BGPO_K_ELL));
  BGPO_TRY(launch_target_logit(ws, dm.d, s));
  BGPO_TRY(tm.end());
  BGPO_TRY(tm.begin(BGPO_K_FWD));
  BGPO_TRY(launch_gemm_fwd(ws, dm.d, dm.V, grid, store_u, s));
  BGPO_TRY(tm.end());
  BGPO_TRY(tm.begin(BGPO_K_ELL));
  BGPO_TRY(launch_combine_rows(ws, dm.V, s));
  BGPO_TRY(launch_seq_terms(ws, dm.B, dm.n_t, j0, adv, ell_old, loss_scale, ell, g, loss, flags,
                            backward, p->bound, dbar, s));
  BGPO_TRY(tm.end(2));
  return BGPO_OK;
}

static int device_grid(int* grid) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return BGPO_ERR_HIP;
  *grid = gemm_grid(dev);
  return BGPO_OK;
}

}  // namespace bgpo

using namespace bgpo;

extern "C" {

int bgpo_version(void) { return (3 << 16) | 1; }

const char* bgpo_status_string(int status) {
  switch (status) {
    case BGPO_OK: return "BGPO_OK";
    case BGPO_ERR_INVALID_ARG: return "BGPO_ERR_INVALID_ARG: invalid argument";
    case BGPO_ERR_WORKSPACE: return "BGPO_ERR_WORKSPACE: workspace missing, misaligned or too small";
    case BGPO_ERR_HIP: return "BGPO_ERR_HIP: a HIP runtime call failed";
    case BGPO_ERR_UNSUPPORTED: return "BGPO_ERR_UNSUPPORTED: shape outside the supported set";
    case BGPO_ERR_BUDGET: return "BGPO_ERR_BUDGET: no workspace layout fits the workspace budget";
    default: return "unknown bgpo status";
  }
}

int bgpo_workspace_size(const bgpo_problem* prob, size_t* bytes) {
  Plan pl;
  const int st = plan_problem(prob, &pl);
  if (st != BGPO_OK) return st;
  if (!bytes) return BGPO_ERR_INVALID_ARG;
  *bytes = workspace_layout(dims_of(prob), pl, nullptr, nullptr, nullptr);
  return BGPO_OK;
}

int bgpo_workspace_plan(const bgpo_problem* prob, bgpo_plan_info* info) {
  Plan pl;
  const int st = plan_problem(prob, &pl);
  if (st != BGPO_OK) return st;
  if (!info) return BGPO_ERR_INVALID_ARG;
  Workspace w;
  info->workspace_bytes = workspace_layout(dims_of(prob), pl, nullptr, &w, nullptr);
  info->samples_per_unit = (int32_t)w.G;
  info->dw_batch = (int32_t)w.dw_batch;
  info->dx_splits = (int32_t)w.n_split;
  info->vocab_chunk = (int32_t)w.chunk;
  info->w_copy = pl.w_copy;
  return BGPO_OK;
}

int bgpo_sample_masks(const bgpo_problem* prob, const uint8_t* resp_mask, int32_t j, int32_t* idx,
                      int32_t* n_masked, float* t_out, void* stream) {
  Plan pl;
  const int st = plan_problem(prob, &pl);
  if (st != BGPO_OK) return st;
  if (!resp_mask || !idx || !n_masked || j < 0 || j >= prob->n_t) return BGPO_ERR_INVALID_ARG;
  if (launch_mask_compact(resp_mask, nullptr, prob->B, prob->L, prob->n_t, j, 0, prob->t_mode,
                          prob->seed, prob->seq_id_base, nullptr, idx, n_masked, 1, t_out, 1,
                          prob->V, nullptr, DxPlan{1, 1, 1, 1}, nullptr, false,
                          (hipStream_t)stream) != hipSuccess)
    return BGPO_ERR_HIP;
  return BGPO_OK;
}

static bool aligned16(const void* p) { return ((uintptr_t)p & 15) == 0; }

static int check_workspace(const bgpo_problem* prob, const Plan& pl, void* workspace,
                           size_t ws_bytes) {
  if (!workspace || ((uintptr_t)workspace % 256) != 0) return BGPO_ERR_WORKSPACE;
  if (ws_bytes < workspace_layout(dims_of(prob), pl, nullptr, nullptr, nullptr))
    return BGPO_ERR_WORKSPACE;
  return BGPO_OK;
}

// [B, n_t] doubles at a and b share a byte
static bool overlaps(const double* a, const double* b, int64_t n) {
  const uintptr_t pa = (uintptr_t)a, pb = (uintptr_t)b, len = (uintptr_t)n * sizeof(double);
  return pa < pb + len && pb < pa + len;
}

}  // extern "C"

namespace bgpo {

// the gradient part of a unit once its scales are known.  Stored mode: the
// forward kept the exponentials; the row factors, the target entries and the
// scaled H_c^T columns make them dZ (up to the row factor, applied to the dX
// rows in the reduction), then one dX GEMM over the whole vocabulary; the
// unit's dZ rows and H_c^T columns are left for the dW GEMM of its batch.
// Recompute mode: per
// vocabulary chunk, the chunk's logits -> its dZ, dX partials accumulated,
// dW[:, chunk] accumulated.  Then each sample's rows are added into dX in
// sample order (with the norm backward).  W: the caller's W_head (bf16
// inputs), read by the dX GEMM when the plan keeps no slab-major copy.
static int unit_backward(const Workspace& ws, const Act& act, int j0, int j_begin,
                         const uint16_t* W, float* dX, float* dgamma, float* dW,
                         const Dims& dm, int grid, Timer& tm, hipStream_t s) {
  if (!ws.chunk) {
    BGPO_TRY(tm.begin(BGPO_K_SOFTMAX_GRAD));
    BGPO_TRY(launch_grad_scale(ws, dm.d, dm.V, s));
    BGPO_TRY(tm.end(3));
    BGPO_TRY(tm.begin(BGPO_K_DX));
    BGPO_TRY(launch_gemm_dx(ws, W, dm.d, dm.V, grid, s));
    BGPO_TRY(tm.end());
  } else {
    for (int v0 = 0; v0 < dm.V; v0 += (int)ws.chunk) {
      const int width = (int)std::min<int64_t>(ws.chunk, dm.V - v0);
      BGPO_TRY(tm.begin(BGPO_K_RECOMPUTE));
      BGPO_TRY(launch_gemm_recompute(ws, dm.d, v0, width, grid, s));
      BGPO_TRY(tm.end());
      BGPO_TRY(tm.begin(BGPO_K_DX));
      BGPO_TRY(launch_gemm_dx_chunk(ws, W, dm.d, dm.V, v0, width, v0 == 0, grid, s));
      BGPO_TRY(tm.end());
      BGPO_TRY(tm.begin(BGPO_K_DW));
      BGPO_TRY(launch_gemm_dw_chunk(ws, dW, dm.d, dm.V, v0, width, grid, s));
      BGPO_TRY(tm.end());
    }
  }
  BGPO_TRY(tm.begin(BGPO_K_DX_REDUCE));
  for (int gs = 0; gs < ws.g_used; ++gs) {
    const int j = j0 + gs;
    float* dXj = dX + (int64_t)(j - j_begin) * act.stride;
    if (act.gamma)
      BGPO_TRY(launch_dx_reduce_rmsnorm(ws, gs, act.at(j), act.f32, act.gamma, dXj, dgamma, dm.d,
                                        s));
    else
      BGPO_TRY(launch_dx_reduce(ws, gs, dXj, dm.d, s));
  }
  BGPO_TRY(tm.end(ws.g_used * (act.gamma ? 3 : 1)));   // the norm backward is 3 kernels
  return BGPO_OK;
}

// The exact objective with every sample's state retained (the way an
// implementation that keeps all n_t computational graphs works): each
// forward runs once and keeps its exponentials, the mean log-ratio is formed,
// then every sample's gradient comes from its kept state; memory grows with
// n_t.  The units are those of the two-pass mode, each with its own state.
static int bwd_retained(const bgpo_problem* prob, const Plan& pl, const Act& act,
                        const void* W_head, const int32_t* targets, const uint8_t* resp_mask,
                        const float* adv, const double* ell_old, double loss_scale, float* dX,
                        float* dgamma, float* dW, double* ell, double* g, double* loss,
                        int32_t* n_masked, float* t_out, int32_t* status_flags, void* workspace,
                        int grid, Timer& tm, hipStream_t s) {
  const Dims dm = dims_of(prob);
  Workspace ws;
  workspace_layout(dm, pl, workspace, &ws, nullptr);
  const int G = (int)ws.G, n_units = (int)ws.dw_batch;
  std::vector<Workspace> U(n_units);
  workspace_layout(dm, pl, workspace, nullptr, U.data());
  BGPO_TRY(tm.begin(BGPO_K_TRANSPOSE_W));
  BGPO_TRY(launch_transpose_w(W_head, act.f32, ws.WT, ws.Wk, dm.d, dm.V, s));
  BGPO_TRY(tm.end());
  for (int u = 0; u < n_units; ++u) {
    const int j0 = u * G, n_s = std::min(G, dm.n_t - j0);
    const int st = run_forward_unit(prob, U[u], tm, grid, j0, n_s, act, targets, resp_mask,
                                    nullptr, nullptr, 0.0, ell, nullptr, nullptr, n_masked, t_out,
                                    status_flags, false, true, u ? U[u - 1].unit() : nullptr,
                                    nullptr, s);
    if (st != BGPO_OK) return st;
  }
  const double* dbar = nullptr;
  if (ell_old) {
    BGPO_TRY(tm.begin(BGPO_K_ELL));
    BGPO_TRY(launch_mean_ratio(ell, ell_old, dm.B, dm.n_t, ws.dbar, s));
    BGPO_TRY(tm.end());
    dbar = ws.dbar;
  }
  for (int u = 0; u < n_units; ++u) {
    const int j0 = u * G;
    BGPO_TRY(tm.begin(BGPO_K_ELL));
    BGPO_TRY(launch_seq_terms(U[u], dm.B, dm.n_t, j0, adv, ell_old, loss_scale, ell, g, loss,
                              status_flags, true, prob->bound, dbar, s));
    BGPO_TRY(tm.end());
    const int st = unit_backward(U[u], act, j0, 0, static_cast<const uint16_t*>(W_head), dX,
                                 dgamma, dW, dm, grid, tm, s);
    if (st != BGPO_OK) return st;
  }
  BGPO_TRY(tm.begin(BGPO_K_DW));
  BGPO_TRY(launch_gemm_dw(U[n_units - 1], dW, dm.d, dm.V, grid, s));
  BGPO_TRY(tm.end());
  return BGPO_OK;
}

static bool aligned_inputs(const Act& act, const void* W_head) {
  return aligned16(act.x) && aligned16(W_head) && (!act.gamma || aligned16(act.gamma));
}

static int elbo_fwd_impl(const bgpo_problem* prob, const Act& act, const void* W_head,
                         const int32_t* targets, const uint8_t* resp_mask, double* ell,
                         int32_t* n_masked, float* t_out, void* workspace, size_t ws_bytes,
                         void* stream, bgpo_timing* prof) {
  Plan pl;
  int st = plan_problem(prob, &pl);
  if (st != BGPO_OK) return st;
  if (!act.x || !W_head || !targets || !resp_mask || !ell || !n_masked) return BGPO_ERR_INVALID_ARG;
  if (!aligned_inputs(act, W_head)) return BGPO_ERR_INVALID_ARG;
  if ((st = check_workspace(prob, pl, workspace, ws_bytes)) != BGPO_OK) return st;
  if (prob->j_count == 0) return BGPO_OK;
  hipStream_t s = (hipStream_t)stream;
  Workspace ws;
  // the layout the workspace was checked against (with retain_samples the
  // first unit's state and the shared buffers; one unit at a time)
  workspace_layout(dims_of(prob), pl, workspace, &ws, nullptr);
  int grid = 0;
  if ((st = device_grid(&grid)) != BGPO_OK) return st;
  Timer tm(prof, s);
  BGPO_TRY(tm.begin(BGPO_K_TRANSPOSE_W));
  BGPO_TRY(launch_transpose_w(W_head, act.f32, ws.WT, nullptr, prob->d, prob->V, s));
  BGPO_TRY(tm.end());
  const int j_end = prob->j_begin + prob->j_count;
  for (int j0 = prob->j_begin; j0 < j_end; j0 += (int)ws.G) {
    const int n_s = std::min<int>(j_end - j0, (int)ws.G);
    st = run_forward_unit(prob, ws, tm, grid, j0, n_s, act, targets, resp_mask, nullptr, nullptr,
                          0.0, ell, nullptr, nullptr, n_masked, t_out, nullptr, false, false,
                          nullptr, nullptr, s);
    if (st != BGPO_OK) return st;
  }
  BGPO_TRY(tm.finish());
  return BGPO_OK;
}

// dX (and dgamma with the norm) are per sample at dX + (j - j_begin) * stride.
static int elbo_bwd_impl(const bgpo_problem* prob, const Act& act, const void* W_head,
                         const int32_t* targets, const uint8_t* resp_mask, const float* adv,
                         const double* ell_old, double loss_scale, float* dX, float* dgamma,
                         float* dW, double* ell, double* g, double* loss, int32_t* n_masked,
                         float* t_out, int32_t* status_flags, void* workspace, size_t ws_bytes,
                         void* stream, bgpo_timing* prof) {
  Plan pl;
  int st = plan_problem(prob, &pl);
  if (st != BGPO_OK) return st;
  if (!act.x || !W_head || !targets || !resp_mask || !adv || !dX || !dW || !ell || !g || !loss ||
      !n_masked || !isfinite(loss_scale) || (act.gamma && !dgamma))
    return BGPO_ERR_INVALID_ARG;
  if (!aligned_inputs(act, W_head) || !aligned16(dX) || !aligned16(dW))
    return BGPO_ERR_INVALID_ARG;
  // l is written before l_old is read (per response, and in the exact mode's
  // first pass for every sample): l_old must be a buffer of its own
  const int64_t nbt = (int64_t)prob->B * prob->n_t;
  if (ell_old && (overlaps(ell_old, ell, nbt) || overlaps(ell_old, g, nbt)))
    return BGPO_ERR_INVALID_ARG;
  if ((st = check_workspace(prob, pl, workspace, ws_bytes)) != BGPO_OK) return st;
  const bool exact = prob->bound == BGPO_BOUND_EXACT;
  if (exact && (prob->j_begin != 0 || prob->j_count != prob->n_t)) return BGPO_ERR_INVALID_ARG;
  if (prob->j_count == 0) return BGPO_OK;
  hipStream_t s = (hipStream_t)stream;
  const Dims dm = dims_of(prob);
  int grid = 0;
  if ((st = device_grid(&grid)) != BGPO_OK) return st;
  Timer tm(prof, s);
  if (prob->retain_samples) {
    st = bwd_retained(prob, pl, act, W_head, targets, resp_mask, adv, ell_old, loss_scale, dX,
                      dgamma, dW, ell, g, loss, n_masked, t_out, status_flags, workspace, grid, tm,
                      s);
    if (st != BGPO_OK) return st;
    BGPO_TRY(tm.finish());
    return BGPO_OK;
  }
  Workspace ws;
  workspace_layout(dm, pl, workspace, &ws, nullptr);
  BGPO_TRY(tm.begin(BGPO_K_TRANSPOSE_W));
  BGPO_TRY(launch_transpose_w(W_head, act.f32, ws.WT, ws.Wk, dm.d, dm.V, s));
  BGPO_TRY(tm.end());
  // exact objective off-policy: a forward pass over every sample gives the
  // mean log-ratio, which scales every sample's gradient (on-policy it is 0)
  const double* dbar = nullptr;
  if (exact && ell_old) {
    for (int j0 = 0; j0 < prob->n_t; j0 += (int)ws.G) {
      const int n_s = std::min<int>(prob->n_t - j0, (int)ws.G);
      st = run_forward_unit(prob, ws, tm, grid, j0, n_s, act, targets, resp_mask, nullptr, nullptr,
                            0.0, ell, nullptr, nullptr, n_masked, t_out, status_flags, false,
                            false, nullptr, nullptr, s);
      if (st != BGPO_OK) return st;
    }
    BGPO_TRY(tm.begin(BGPO_K_ELL));
    BGPO_TRY(launch_mean_ratio(ell, ell_old, dm.B, dm.n_t, ws.dbar, s));
    BGPO_TRY(tm.end());
    dbar = ws.dbar;
  }
  const int j_end = prob->j_begin + prob->j_count;
  const bool store_u = !ws.chunk;   // stored mode keeps the forward's exponentials
  int in_batch = 0;        // units already in the current dW batch
  int prev_used = 0;       // samples of the previous unit (its record is meta[prev_used - 1])
  for (int j0 = prob->j_begin; j0 < j_end; j0 += (int)ws.G) {
    const int n_s = std::min<int>(j_end - j0, (int)ws.G);
    // a unit after the first of its batch puts its dZ rows / H_c^T columns
    // after the previous unit's (whose last record the first mask launch reads
    // before any record is rewritten)
    const SampleMeta* prev = in_batch ? ws.meta + (prev_used - 1) : nullptr;
    st = run_forward_unit(prob, ws, tm, grid, j0, n_s, act, targets, resp_mask, adv, ell_old,
                          loss_scale, ell, g, loss, n_masked, t_out, status_flags, true, store_u,
                          prev, dbar, s);
    if (st != BGPO_OK) return st;
    st = unit_backward(ws, act, j0, prob->j_begin, static_cast<const uint16_t*>(W_head), dX,
                       dgamma, dW, dm, grid, tm, s);
    if (st != BGPO_OK) return st;
    prev_used = n_s;
    // stored mode: one dW GEMM per batch of units, K over all their rows (the
    // recompute mode accumulated dW chunk by chunk)
    if (!ws.chunk && (++in_batch == (int)ws.dw_batch || j0 + n_s >= j_end)) {
      BGPO_TRY(tm.begin(BGPO_K_DW));
      BGPO_TRY(launch_gemm_dw(ws, dW, dm.d, dm.V, grid, s));
      BGPO_TRY(tm.end());
      in_batch = 0;
    }
  }
  BGPO_TRY(tm.finish());
  return BGPO_OK;
}

static Act act_of(const bgpo_problem* p, const void* x, const float* gamma) {
  return Act{x, p && p->in_dtype == BGPO_F32, gamma, p ? p->norm_eps : 0.f,
             p ? p->sample_stride : 0, p ? p->j_begin : 0};
}

}  // namespace bgpo

extern "C" {

int bgpo_elbo_fwd(const bgpo_problem* prob, const void* hidden, const void* W_head,
                  const int32_t* targets, const uint8_t* resp_mask, double* ell,
                  int32_t* n_masked, float* t_out, void* workspace, size_t ws_bytes, void* stream,
                  bgpo_timing* prof) {
  return elbo_fwd_impl(prob, act_of(prob, hidden, nullptr), W_head, targets, resp_mask, ell,
                       n_masked, t_out, workspace, ws_bytes, stream, prof);
}

int bgpo_elbo_bwd_accumulate(const bgpo_problem* prob, const void* hidden,
                             const void* W_head, const int32_t* targets,
                             const uint8_t* resp_mask, const float* adv, const double* ell_old,
                             double loss_scale, float* dX, float* dW, double* ell, double* g,
                             double* loss, int32_t* n_masked, float* t_out, int32_t* status_flags,
                             void* workspace, size_t ws_bytes, void* stream, bgpo_timing* prof) {
  return elbo_bwd_impl(prob, act_of(prob, hidden, nullptr), W_head, targets, resp_mask, adv,
                       ell_old, loss_scale, dX, nullptr, dW, ell, g, loss, n_masked, t_out,
                       status_flags, workspace, ws_bytes, stream, prof);
}

int bgpo_elbo_fwd_rmsnorm(const bgpo_problem* prob, const void* x, const float* norm_weight,
                          const void* W_head, const int32_t* targets,
                          const uint8_t* resp_mask, double* ell, int32_t* n_masked, float* t_out,
                          void* workspace, size_t ws_bytes, void* stream, bgpo_timing* prof) {
  if (!norm_weight) return BGPO_ERR_INVALID_ARG;
  return elbo_fwd_impl(prob, act_of(prob, x, norm_weight), W_head, targets, resp_mask, ell,
                       n_masked, t_out, workspace, ws_bytes, stream, prof);
}

int bgpo_elbo_bwd_accumulate_rmsnorm(const bgpo_problem* prob, const void* x,
                                     const float* norm_weight, const void* W_head,
                                     const int32_t* targets, const uint8_t* resp_mask,
                                     const float* adv, const double* ell_old, double loss_scale,
                                     float* dx, float* d_norm_weight, float* dW, double* ell,
                                     double* g, double* loss, int32_t* n_masked, float* t_out,
                                     int32_t* status_flags, void* workspace, size_t ws_bytes,
                                     void* stream, bgpo_timing* prof) {
  if (!norm_weight || !d_norm_weight) return BGPO_ERR_INVALID_ARG;
  return elbo_bwd_impl(prob, act_of(prob, x, norm_weight), W_head, targets, resp_mask, adv,
                       ell_old, loss_scale, dx, d_norm_weight, dW, ell, g, loss, n_masked, t_out,
                       status_flags, workspace, ws_bytes, stream, prof);
}

}  // extern "C"

// ---------------------------------------------------------------------------
// The backward without a caller workspace: its workspace is a static device
// array of kScratchBytes (each device the library runs on holds its own copy
// until the process ends).  The array's name is a host-side stand-in, so the
// device address of each device's copy is looked up once, with that device
// current, and only that address is handed to the kernels.
namespace bgpo {

constexpr size_t kScratchBytes = size_t(128) << 20;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
static std::mutex g_scratch_mu;
static void* g_scratch_ptr[kMaxDevices];

// device address of the current device's scratch array (NULL on failure)
static void* scratch_of_current_device() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) return nullptr;
    g_scratch_ptr[dev] = ptr;
  }
  return g_scratch_ptr[dev];
}

}  // namespace bgpo

extern "C" size_t bgpo_noalloc_scratch_bytes(void) { return bgpo::kScratchBytes; }

extern "C" int bgpo_elbo_bwd_accumulate_noalloc(
    const bgpo_problem* prob, const void* hidden, const void* W_head, const int32_t* targets,
    const uint8_t* resp_mask, const float* adv, const double* ell_old, double loss_scale,
    float* dX, float* dW, double* ell, double* g, double* loss, int32_t* n_masked, float* t_out,
    int32_t* status_flags, void* stream) {
  using namespace bgpo;
  if (!prob) return BGPO_ERR_INVALID_ARG;
  if (prob->retain_samples) return BGPO_ERR_INVALID_ARG;   // memory grows with n_t
  // the problem's layout within the scratch array: its own budget if smaller
  bgpo_problem p = *prob;
  if (p.ws_budget == 0 || p.ws_budget > kScratchBytes) p.ws_budget = kScratchBytes;
  Plan pl;
  const int st = plan_problem(&p, &pl);
  if (st != BGPO_OK) return st;   // BGPO_ERR_BUDGET: the problem needs more than the scratch
  void* ws = scratch_of_current_device();
  if (!ws) return BGPO_ERR_HIP;
  return elbo_bwd_impl(&p, act_of(&p, hidden, nullptr), W_head, targets, resp_mask, adv, ell_old,
                       loss_scale, dX, nullptr, dW, ell, g, loss, n_masked, t_out, status_flags,
                       ws, kScratchBytes, stream, nullptr);
}

// ---- test hook: the multi-block mask passes at any size ----
extern "C" size_t bgpo_test_mask_scratch_bytes(const bgpo_problem* prob) {
  return prob ? bgpo::mask_scratch_bytes(prob->B, prob->L) : 0;
}

extern "C" int bgpo_test_mask_multiblock(const bgpo_problem* prob, const uint8_t* resp_mask,
                                         int32_t j, int32_t* idx, int32_t* n_masked,
                                         float* t_out, void* scratch, size_t scratch_bytes,
                                         void* stream) {
  using namespace bgpo;
  Plan pl;
  const int st = plan_problem(prob, &pl);
  if (st != BGPO_OK) return st;
  if (!resp_mask || !idx || !n_masked || j < 0 || j >= prob->n_t) return BGPO_ERR_INVALID_ARG;
  if (!scratch || ((uintptr_t)scratch % 256) != 0 ||
      scratch_bytes < mask_scratch_bytes(prob->B, prob->L))
    return BGPO_ERR_WORKSPACE;
  if (launch_mask_compact(resp_mask, nullptr, prob->B, prob->L, prob->n_t, j, 0, prob->t_mode,
                          prob->seed, prob->seq_id_base, nullptr, idx, n_masked, 1, t_out, 1,
                          prob->V, nullptr, DxPlan{1, 1, 1, 1}, scratch, true,
                          (hipStream_t)stream) != hipSuccess)
    return BGPO_ERR_HIP;
  return BGPO_OK;
}
