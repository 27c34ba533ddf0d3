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

// Device-resident per-sample bookkeeping written by the mask kernel.
struct SampleMeta {
  int32_t n_rows;      // N_j: masked positions in this sample (all responses)
  int32_t n_rows_pad;  // N_j rounded up to kRowPad
  int32_t col_off;     // first column of this sample in H_c^T / dZ^T
  int32_t col_end;     // col_off + N_j rounded up to 64: K of the batched dW GEMM
  int32_t dx_split;    // vocabulary splits of this sample's dX GEMM
  int32_t dx_kslab;    // 64-wide vocabulary slabs per split
  int32_t pad[58];
};

// What the mask kernel needs to choose the dX split of a sample (the split
// count that best fills the persistent grid for the sample's row count).
struct DxPlan {
  int kslabs;      // V / 64
  int col_tiles;   // d / 256
  int grid;        // workgroups of the persistent GEMM grid
  int s_max;       // splits the partial buffer holds
};

// Views into the caller's workspace.
struct Workspace {
  SampleMeta* meta;
  int32_t* idx;        // [P]          masked flat positions, ascending
  int32_t* row_tgt;    // [NP]         target token of each compacted row
  int32_t* row_seq;    // [NP]         response of each compacted row (B for padding)
  int32_t* seg_off;    // [B+1]        first compacted row of each response
  uint32_t* t24;       // [B]          integer timestep of each response
  uint16_t* Hc;        // [NP, d]      gathered masked hidden rows (bf16)
  uint16_t* HcT;       // [d, KT]      the same, transposed; samples of a dW batch side by side
  uint16_t* WT;        // [V, d]       W_head transposed (bf16)
  float* part_m;       // [nvt, NP]    per-vocabulary-slice max (log2 units)
  float* part_s;       // [nvt, NP]    per-vocabulary-slice sum of 2^(z*log2e - max)
  float* ztgt;         // [NP]         target logit
  float* lse2;         // [NP]         log2-sum-exp2 of each row (log2 units)
  float* lp;           // [NP]         log p of the target
  float* row_scale;    // [NP]         gradient scale s of each row (0 for padding)
  double* dbar;        // [B]          mean log-ratio over all samples (exact objective)
  float* inv_rms;      // [NP]         final-RMSNorm 1/rms of each compacted row
  float* gpart;        // [NP/256, d]  dgamma partial sums over 256-row chunks
  uint16_t* dZ;        // [NP, V]      s (softmax - onehot), bf16 (first the fp16 exponentials)
  uint16_t* dZT;       // [V, KT]      the same, transposed; samples of a dW batch side by side
  float* dx_part;      // [S, NP, d]   split-vocabulary partial dX
  int64_t P, NP, nvt;
  int64_t n_split;     // capacity of dx_part in splits (the per-sample count is in meta)
  int64_t dw_batch;    // samples whose dW contributions share one GEMM
  int64_t KT;          // dw_batch * NP: leading dimension of H_c^T and dZ^T
};

struct Dims {
  int B, L, d, V, n_t;
};

// Views into the caller's workspace (base may be NULL: sizes only).
// retain = 0: the state of one sample at a time, dW batches of up to
//             kMaxDwBatch samples; the size does not depend on n_t.
// retain = 1: the state of every one of the n_t samples is kept
//             (samples[0 .. n_t), each with its own meta, rows, partials, H_c
//             and dZ; H_c^T / dZ^T hold all samples' columns; one dW batch).
size_t workspace_layout(const Dims& dm, int retain, void* base, Workspace* ws,
                        Workspace* samples);

// ---- launchers (return hipSuccess or the launch error) ----
hipError_t launch_transpose_w(const uint16_t* W, uint16_t* WT, int d, int V, hipStream_t s);
hipError_t launch_mask_compact(const uint8_t* resp, const int32_t* targets, int B, int L, int n_t, int j,
                               int t_mode, uint64_t seed, uint32_t seq_base, int32_t* idx,
                               int32_t* row_tgt, int32_t* row_seq, int32_t* seg_off, uint32_t* t24,
                               SampleMeta* meta, int32_t* n_masked_out, int nm_stride,
                               float* t_out, int t_stride, int row_cap, int V,
                               const SampleMeta* prev, const DxPlan& plan, hipStream_t s);
hipError_t launch_row_rms(const uint16_t* x, const Workspace& ws, int d, float eps, hipStream_t s);
hipError_t launch_gather(const uint16_t* hidden, const float* gamma, const Workspace& ws, int d,
                         hipStream_t s);
hipError_t launch_gemm_fwd(const Workspace& ws, int d, int V, int grid, bool store_u,
                           hipStream_t s);
hipError_t launch_target_logit(const Workspace& ws, int d, hipStream_t s);
hipError_t launch_combine_rows(const Workspace& ws, int V, hipStream_t s);
hipError_t launch_seq_terms(const Workspace& ws, int B, int n_t, int j, const float* adv,
                            const double* ell_old, double loss_scale, double* ell, double* g,
                            double* loss, int32_t* flags, bool backward, int bound,
                            const double* dbar, hipStream_t s);
hipError_t launch_mean_ratio(const double* ell, const double* ell_old, int B, int n_t,
                             double* dbar, hipStream_t s);
hipError_t launch_softmax_grad(const Workspace& ws, int V, hipStream_t s);
hipError_t launch_gemm_dx(const Workspace& ws, const uint16_t* W, int d, int V, int grid,
                          hipStream_t s);
hipError_t launch_dx_reduce(const Workspace& ws, float* dX, int d, hipStream_t s);
hipError_t launch_dx_reduce_rmsnorm(const Workspace& ws, const uint16_t* x, const float* gamma,
                                    float* dx, float* dgamma, int d, hipStream_t s);
hipError_t launch_gemm_dw(const Workspace& ws, float* dW, int d, int V, int grid, hipStream_t s);

int gemm_grid(int device);  // persistent grid size of the GEMM kernels on `device`

}  // namespace bgpo
