// Host-side declarations shared by the translation units of libbgpo.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace bgpo {

// Rows of the compacted masked-position list are padded to a multiple of
// this (the row tile of the LM-head GEMMs); padded rows carry zeros.
constexpr int kRowPad = 256;
// Vocabulary slice of one log-sum-exp partial (the M extent of one wave of the
// LM-head GEMM).
constexpr int kVocabTile = 128;

constexpr int kFlagNonfinite = 1;   // BGPO_FLAG_NONFINITE

// Stored backward: the forward keeps each row's exponentials against one
// reference per row, R2 = z_target log2e + kExpRef (log2 units), so that
// dZ = f (u - onehot 2^(lse2 - R2)) with one factor f = s 2^(R2 - lse2) per
// row.  A row whose log2-sum-exp exceeds R2 by more than kExpRange (the
// target's log2 probability below -(kExpRef + kExpRange)) would leave the
// exponent range of the operands; its exponentials are recomputed against
// R2 = lse2 after the forward.
constexpr float kExpRef = 60.f;
constexpr float kExpRange = 64.f;
__host__ __device__ inline float exp_reference(float ztgt) { return ztgt * 1.4426950408889634f + kExpRef; }

// Column capacity of H_c^T, row capacity of the stored dZ (the rows of a dW
// batch; the offsets of the sample records are 32-bit).
constexpr int64_t kMaxColumns = int64_t(1) << 30;

// Rows per slab of the stored dZ: KT plus this padding, so that the slabs of
// one vocabulary tile (which the dW GEMM reads side by side) do not lie a
// power of two apart.
constexpr int64_t kDzPadRows = 64;

// K-slab-major layout of a bf16 operand with R rows per slab: element (r, k)
// at ((k / 64) R + r) 64 + k % 64 (the GEMMs' operand layout: one 64-deep
// slab of 256 consecutive rows is 32 KB of contiguous memory).
__host__ __device__ inline int64_t slab_index(int64_t R, int64_t r, int64_t k) {
  return ((k >> 6) * R + r) * 64 + (k & 63);
}

// Device-resident bookkeeping written by the mask kernel, one record per
// sample.  Samples are processed in units of up to G consecutive samples whose
// masked rows sit back to back in one row space (the LM-head GEMMs and the row
// kernels run once per unit); the unit-level fields are cumulative, so the
// record of the unit's last sample describes the whole unit.
struct SampleMeta {
  int32_t n_rows;      // masked rows of the unit up to and including this sample
  int32_t n_rows_pad;  // n_rows rounded up to kRowPad
  int32_t col_off;     // first column of the unit in H_c^T (and row in the stored dZ)
  int32_t col_end;     // col_off + n_rows rounded up to 64: K of the dW GEMM
  int32_t dx_split;    // vocabulary splits of the unit's dX GEMM
  int32_t dx_kslab;    // 64-wide vocabulary slabs per split
  int32_t s_rows;      // N_j: masked rows of this sample (all responses)
  int32_t s_row_off;   // first row of this sample in the unit's row space
  int32_t pad[56];
};

// What the mask kernel needs to choose the dX split of a unit (the split
// count that best fills the persistent grid for the unit's row count).
struct DxPlan {
  int kslabs;      // V / 64
  int col_tiles;   // d / 256
  int grid;        // workgroups of the persistent GEMM grid
  int s_max;       // splits the partial buffer holds
};

// Views into the caller's workspace: the state of one unit of G samples
// (RP = G * NP rows) and the buffers shared by all units.
struct Workspace {
  SampleMeta* meta;    // [G]          one record per sample of the unit
  int32_t* idx;        // [G*P]        masked flat positions, per sample ascending
  int32_t* row_tgt;    // [RP]         target token of each compacted row
  int32_t* row_seq;    // [RP]         g*B + b of each row (sample g of the unit, response b)
  int32_t* seg_off;    // [G*(B+1)]    first row of each (sample, response), unit row space
  uint32_t* t24;       // [G*B]        integer timestep of each (sample, response)
  float* seq_scale;    // [G*B]        gradient scale s of each (sample, response)
  // (slab-major: a matrix with R rows per slab and K columns, see slab_index)
  uint16_t* Hc;        // [RP rows, d] gathered masked hidden rows (bf16), slab-major
  uint16_t* HcT;       // [d rows, KT] the same, transposed, units of a dW batch side by side,
                       // slab-major
  uint16_t* WT;        // [V, d]       W_head transposed (bf16), row-major
  uint16_t* Wk;        // [d rows, V]  W_head in bf16, slab-major: the dX GEMM's A operand
                       // (NULL without Plan::w_copy)
  float* part_m;       // [nvt, RP]    per-vocabulary-slice max (log2 units)
  float* part_s;       // [nvt, RP]    per-vocabulary-slice sum of 2^(z*log2e - max)
  float* ztgt;         // [RP]         target logit
  float* lse2;         // [RP]         log2-sum-exp2 of each row (log2 units)
  float* lp;           // [RP]         log p of the target
  float* row_scale;    // [RP]         gradient scale s of each row (0 for padding)
  float* row_f;        // [RP]         stored backward: dZ row factor s 2^(R2 - lse2) (0 for padding)
  uint8_t* row_bad;    // [RP]         stored backward: row recomputed against R2 = lse2
  double* dbar;        // [B]          mean log-ratio over all samples (exact objective)
  float* inv_rms;      // [RP]         final-RMSNorm 1/rms of each compacted row
  void* mask_scratch;  // mask_scratch_bytes(B, L): the multi-block mask passes
  float* gpart;        // [NP/256, d]  dgamma partial sums over 256-row chunks of a sample
  uint16_t* dZ;        // stored mode: [KT rows, V] the forward's bf16 exponentials against
                       // the row's reference, i.e. s (softmax - onehot) up to the row factor
                       // (target entries rewritten), the units of a dW batch one after the
                       // other (unit rows from its col_off); recompute mode: [RP rows,
                       // chunk], one vocabulary chunk's s (softmax - onehot); slab-major
  float* dx_part;      // [S, RP, d]   split-vocabulary partial dX
  int64_t P, NP, nvt;
  int64_t G;           // samples per unit
  int64_t RP;          // G * NP: row capacity of a unit
  int64_t n_split;     // capacity of dx_part in splits (the unit's count is in its meta)
  int64_t dw_batch;    // units whose dW contributions share one GEMM
  int64_t KT;          // dw_batch * RP: columns of H_c^T, rows of the stored dZ
  int64_t ldz;         // rows per slab of dZ: KT + kDzPadRows (stored), RP (recompute)
  int64_t chunk;       // 0: stored exponentials; > 0: recompute backward, vocabulary chunk width
  int g_used;          // samples in the current unit (host side; its record meta[g_used - 1]
                       // describes the unit)
  const SampleMeta* unit() const { return meta + (g_used - 1); }
};

struct Dims {
  int B, L, d, V, n_t;
};

// How a problem uses its workspace, chosen from the shapes, the input type and
// the budget (never from n_t, except the unit count of the retained mode).
struct Plan {
  int64_t G;          // samples per unit
  int64_t dw_batch;   // units per dW GEMM (stored mode)
  int64_t n_split;    // capacity of the dX split partials, in splits
  int64_t chunk;      // 0: stored exponentials; > 0: recompute in vocabulary chunks of this width
  int retain;         // every unit keeps its own state (memory grows with n_t)
  int w_copy;         // keep the slab-major bf16 copy of W_head that the dX GEMM reads
                      // (else it reads the caller's bf16 W_head row-major; always 1 for
                      // fp32 inputs)
};

// Views into the caller's workspace for plan `pl` (base may be NULL: sizes
// only).
// retain = 0: the state of one unit of G samples at a time, dw_batch units
//             per dW GEMM; the size does not depend on n_t.
// retain = 1: the same units (G capped at n_t), each keeping its own state
//             (units[0 .. ceil(n_t / G)): meta, rows, partials, H_c; H_c^T
//             and dZ hold all units' columns and rows; one dW batch), so
//             memory grows with n_t.
size_t workspace_layout(const Dims& dm, const Plan& pl, void* base, Workspace* ws,
                        Workspace* units);

// ---- launchers (return hipSuccess or the launch error) ----
// W_head -> W^T (bf16, row-major) and W (bf16, slab-major with d rows per
// slab); fp32 W (f32) is rounded to bf16 as it is read
hipError_t launch_transpose_w(const void* W, bool f32, uint16_t* WT, uint16_t* Wk, int d, int V,
                              hipStream_t s);
// Mask and compaction of sample j, sample g of its unit: rows go after those of
// the unit's earlier samples (prev = record of sample g - 1); for g = 0, prev
// (may be NULL) is the record of the previous unit of the dW batch, whose
// columns this unit's follow.
hipError_t launch_mask_compact(const uint8_t* resp, const int32_t* targets, int B, int L, int n_t,
                               int j, int g, int t_mode, uint64_t seed, uint32_t seq_base,
                               const Workspace* ws, int32_t* idx_out, int32_t* n_masked_out,
                               int nm_stride, float* t_out, int t_stride, int V,
                               const SampleMeta* prev, const DxPlan& plan, void* scratch,
                               bool force_multi, hipStream_t s);
// scratch bytes the multi-block mask passes need (mask words, block counts and
// offsets, timesteps); with scratch NULL the single-workgroup kernel runs, and
// with scratch the multi-block passes run above 65536 positions (or always,
// with force_multi)
size_t mask_scratch_bytes(int B, int L);
// x / hidden of row r is x + (row_seq[r] / B) * stride (the row's sample in the unit)
// (f32: x / hidden are fp32, rounded to bf16 as they are read)
hipError_t launch_row_rms(const void* x, bool f32, int64_t stride, int B, const Workspace& ws,
                          int d, float eps, hipStream_t s);
hipError_t launch_gather(const void* hidden, bool f32, int64_t stride, int B, const float* gamma,
                         const Workspace& ws, int d, hipStream_t s);
hipError_t launch_gemm_fwd(const Workspace& ws, int d, int V, int grid, bool store_u,
                           hipStream_t s);
hipError_t launch_target_logit(const Workspace& ws, int d, hipStream_t s);
hipError_t launch_combine_rows(const Workspace& ws, int V, hipStream_t s);
// per-response terms of the unit's samples j0 .. j0 + g_used - 1
hipError_t launch_seq_terms(const Workspace& ws, int B, int n_t, int j0, const float* adv,
                            const double* ell_old, double loss_scale, double* ell, double* g,
                            double* loss, int32_t* flags, bool backward, int bound,
                            const double* dbar, hipStream_t s);
hipError_t launch_mean_ratio(const double* ell, const double* ell_old, int B, int n_t,
                             double* dbar, hipStream_t s);
// stored backward, after the unit's scales: row factors, the target entries of
// dZ, H_c^T scaled by the row factors, and the rows outside the exponent range
// recomputed
hipError_t launch_grad_scale(const Workspace& ws, int d, int V, hipStream_t s);
// (W: the caller's bf16 W_head, read row-major when ws.Wk is NULL)
hipError_t launch_gemm_dx(const Workspace& ws, const uint16_t* W, int d, int V, int grid,
                          hipStream_t s);
// dX of sample g of the unit (its rows only; samples of a unit run one after
// the other, so positions shared between samples are summed in sample order)
hipError_t launch_dx_reduce(const Workspace& ws, int g, float* dX, int d, hipStream_t s);
hipError_t launch_dx_reduce_rmsnorm(const Workspace& ws, int g, const void* x, bool f32,
                                    const float* gamma, float* dx, float* dgamma, int d,
                                    hipStream_t s);
hipError_t launch_gemm_dw(const Workspace& ws, float* dW, int d, int V, int grid, hipStream_t s);
// recompute mode, vocabulary chunk [v0, v0 + width): the chunk's logits from
// W^T and H_c, turned into dZ = s (softmax - onehot) (bf16);
// dX^T partials (+)= W[:, chunk] . dZ^T (first chunk: stored);
// dW[:, chunk] += H_c^T . dZ
hipError_t launch_gemm_recompute(const Workspace& ws, int d, int v0, int width, int grid,
                                 hipStream_t s);
// (W: the caller's bf16 W_head, read row-major when ws.Wk is NULL)
hipError_t launch_gemm_dx_chunk(const Workspace& ws, const uint16_t* W, int d, int V, int v0,
                                int width, bool first, int grid, hipStream_t s);
hipError_t launch_gemm_dw_chunk(const Workspace& ws, float* dW, int d, int V, int v0, int width,
                                int grid, hipStream_t s);

int gemm_grid(int device);  // persistent grid size of the GEMM kernels on `device`

}  // namespace bgpo
