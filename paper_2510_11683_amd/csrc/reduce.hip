// Row and response reductions of the ELBO head:
//   target logit      z[row, y_row] = Hc[row] . W[:, y_row]
//   log-sum-exp       combine the per-vocabulary-tile (max, sum) partials
//   per-response      l = (1/t) sum log p (Eq. per_step_loss), d, g (Eq. g),
//                     loss (Algorithm 1, L_j = -g_j/G) and the gradient scale
//   stored backward   per-row factors of the kept exponentials, their target
//                     entries (the one-hot term), H_c^T scaled by the
//                     factors, and rows outside the exponent range recomputed
//   dX                sum of the split-vocabulary partials, scattered to the
//                     masked positions
// Every reduction runs in a fixed order, so results are bit-reproducible.
#include "common.hpp"
#include "internal.hpp"

namespace bgpo {

// One wave per row: 64 lanes split the d-long dot product (Hc slab-major with
// RP rows per slab: each group of 8 lanes reads one 128-byte slab row).
__global__ __launch_bounds__(256) void k_target_logit(const uint16_t* __restrict__ Hc,
                                                      const uint16_t* __restrict__ WT,
                                                      const int32_t* __restrict__ row_tgt,
                                                      const SampleMeta* __restrict__ meta,
                                                      float* __restrict__ ztgt, int d,
                                                      int64_t RP) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= meta->n_rows) return;
  const uint16_t* w = WT + (int64_t)row_tgt[row] * d;
  float acc = 0.f;
  for (int k = lane * 8; k < d; k += 64 * 8) {
    const uint4 hv = *reinterpret_cast<const uint4*>(Hc + slab_index(RP, row, k));
    const uint4 wv = *reinterpret_cast<const uint4*>(w + k);
    const uint32_t ha[4] = {hv.x, hv.y, hv.z, hv.w}, wa[4] = {wv.x, wv.y, wv.z, wv.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      acc = fmaf(__uint_as_float(ha[e] << 16), __uint_as_float(wa[e] << 16), acc);
      acc = fmaf(__uint_as_float(ha[e] & 0xFFFF0000u), __uint_as_float(wa[e] & 0xFFFF0000u), acc);
    }
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) acc += __shfl_xor(acc, off, 64);
  if (lane == 0) ztgt[row] = acc;
}

hipError_t launch_target_logit(const Workspace& ws, int d, hipStream_t s) {
  k_target_logit<<<(unsigned)(ws.RP / 4), 256, 0, s>>>(ws.Hc, ws.WT, ws.row_tgt, ws.unit(), ws.ztgt,
                                                       d, ws.RP);
  return hipGetLastError();
}

// log-sum-exp of every row from its per-slice (max, sum) partials, and the
// target's log p.  64 rows per workgroup, one per lane, so each load of a
// slice's partials is 64 consecutive floats; the 16 waves take every 16th
// slice, 8 slices' loads in flight at a time, and are combined in LDS in a
// fixed order.
constexpr int kCombineWaves = 16;

__global__ __launch_bounds__(64 * kCombineWaves) void k_combine_rows(
    const float* __restrict__ part_m, const float* __restrict__ part_s,
    const float* __restrict__ ztgt, const SampleMeta* __restrict__ meta,
    float* __restrict__ lse2, float* __restrict__ lp, int nvt, int64_t ldp) {
  __shared__ float sm[kCombineWaves][64], ss[kCombineWaves][64];
  const int lane = threadIdx.x & 63, q = threadIdx.x >> 6;
  const int row = blockIdx.x * 64 + lane;
  const int n_rows = meta->n_rows;
  if (blockIdx.x * 64 >= n_rows) return;
  float m = -INFINITY, sum = 0.f;
  if (row < n_rows) {
    for (int t0 = q; t0 < nvt; t0 += kCombineWaves * 8) {
      float mt[8], st[8];
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        const int t = t0 + kCombineWaves * k;
        mt[k] = t < nvt ? part_m[(int64_t)t * ldp + row] : -INFINITY;
        st[k] = t < nvt ? part_s[(int64_t)t * ldp + row] : 0.f;
      }
#pragma unroll
      for (int k = 0; k < 8; ++k) {
        if (st[k] > 0.f) {
          const float mn = fmaxf(m, mt[k]);
          sum = sum * exp2f(m - mn) + st[k] * exp2f(mt[k] - mn);
          m = mn;
        }
      }
    }
  }
  sm[q][lane] = m;
  ss[q][lane] = sum;
  __syncthreads();
  if (q == 0 && row < n_rows) {
    float M = -INFINITY;
#pragma unroll
    for (int k = 0; k < kCombineWaves; ++k) M = fmaxf(M, sm[k][lane]);
    float S = 0.f;
#pragma unroll
    for (int k = 0; k < kCombineWaves; ++k)
      if (ss[k][lane] > 0.f) S += ss[k][lane] * exp2f(sm[k][lane] - M);
    const float l2 = M + log2f(S);
    lse2[row] = l2;
    lp[row] = ztgt[row] - l2 * kLn2;
  }
}

hipError_t launch_combine_rows(const Workspace& ws, int V, hipStream_t s) {
  k_combine_rows<<<(unsigned)(ws.RP / 64), 64 * kCombineWaves, 0, s>>>(
      ws.part_m, ws.part_s, ws.ztgt, ws.unit(), ws.lse2, ws.lp, (int)ws.nvt, ws.RP);
  return hipGetLastError();
}

// Per-response terms of the samples of a unit.  One workgroup; each wave
// takes (sample, response) segments wave, wave + 16, ...; the loss is then
// summed by one thread over the segments in sample-then-response order.
constexpr int kSeqThreads = 1024;

// The objective's per-sample term g and its derivative dg/dl for
// d = l - l_old:
//   paper (Eq. g):  first-order Taylor bound (1 + d) A / n_t for A >= 0
//                   (Lemma 1), Jensen bound e^d A / n_t for A < 0 (Lemma 2)
//   Taylor only / Jensen only: one of the two for every sign (the ablation of
//                   Table 3)
//   exact:          exp(dbar) A / n_t with dbar the mean of d over all n_t
//                   samples, whose sum is exp(B_theta - B_old) A
//                   (Eq. elbo_ratio); dg/dl_j = exp(dbar) A / n_t
__device__ __forceinline__ void bound_term(double dj, double A, int n_t, int bound, double dbar,
                                           double* gj, double* dg) {
  if (bound == 3) {
    *gj = exp(dbar) * A / n_t;
    *dg = *gj;
  } else if (bound == 1 || (bound == 0 && A >= 0.0)) {
    *gj = (1.0 + dj) * A / n_t;
    *dg = A / n_t;
  } else {
    *gj = exp(dj) * A / n_t;
    *dg = *gj;
  }
}

// Sample g of the unit is sample j0 + g; its response b has rows
// [seg_off[g (B+1) + b], seg_off[g (B+1) + b + 1]) and timestep t24[g B + b].
// The gradient scale of (g, b) goes to seq_scale[g B + b] and from there to
// every row of that response (row_seq[r] = g B + b).
__global__ __launch_bounds__(kSeqThreads) void k_seq_terms(
    const float* __restrict__ lp, const int32_t* __restrict__ seg_off,
    const uint32_t* __restrict__ t24, const int32_t* __restrict__ row_seq,
    const SampleMeta* __restrict__ meta, int B, int n_t, int j0, int n_samples,
    const float* __restrict__ adv, const double* __restrict__ ell_old, double loss_scale,
    double* __restrict__ ell, double* __restrict__ g, double* __restrict__ loss,
    int32_t* __restrict__ flags, float* __restrict__ seq_scale, float* __restrict__ row_scale,
    int backward, int bound, const double* __restrict__ dbar) {
  __shared__ int s_bad;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  if (tid == 0) s_bad = 0;
  __syncthreads();
  const int n_seg = n_samples * B;
  for (int sg = wave; sg < n_seg; sg += kSeqThreads / 64) {
    const int gs = sg / B, b = sg - gs * B, j = j0 + gs;
    const int r0 = seg_off[gs * (B + 1) + b], r1 = seg_off[gs * (B + 1) + b + 1];
    double acc = 0.0;
    for (int r = r0 + lane; r < r1; r += 64) acc += (double)lp[r];
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) acc += __shfl_xor(acc, off, 64);
    if (lane == 0) {
      const double t = (double)t24[gs * B + b] * (1.0 / 16777216.0);
      const double l = acc / t;                                        // Eq. per_step_loss
      const int64_t o = (int64_t)b * n_t + j;
      ell[o] = l;
      if (backward) {
        const double dj = ell_old ? l - ell_old[o] : 0.0;
        double gj, dg;
        bound_term(dj, (double)adv[b], n_t, bound, dbar ? dbar[b] : 0.0, &gj, &dg);
        g[o] = gj;
        const double sc = loss_scale * dg / t;
        seq_scale[gs * B + b] = (float)sc;
        if (!isfinite(l) || !isfinite(gj) || !isfinite(sc) || !isfinite((float)sc)) s_bad = 1;
      } else if (!isfinite(l)) {
        s_bad = 1;
      }
    }
  }
  // g and seq_scale of every segment are written (global memory) before here
  __threadfence_block();
  __syncthreads();
  if (tid == 0) {
    if (backward) {
      double loss_acc = 0.0;
      for (int gs = 0; gs < n_samples; ++gs)
        for (int b = 0; b < B; ++b) loss_acc += -loss_scale * g[(int64_t)b * n_t + j0 + gs];
      loss[0] += loss_acc;
    }
    if (s_bad && flags) atomicOr(flags, kFlagNonfinite);
  }
  if (backward) {
    const int N = meta->n_rows, NPr = meta->n_rows_pad;
    for (int r = tid; r < NPr; r += kSeqThreads) row_scale[r] = r < N ? seq_scale[row_seq[r]] : 0.f;
  }
}

hipError_t launch_seq_terms(const Workspace& ws, int B, int n_t, int j0, const float* adv,
                            const double* ell_old, double loss_scale, double* ell, double* g,
                            double* loss, int32_t* flags, bool backward, int bound,
                            const double* dbar, hipStream_t s) {
  k_seq_terms<<<1, kSeqThreads, 0, s>>>(ws.lp, ws.seg_off, ws.t24, ws.row_seq, ws.unit(), B, n_t,
                                        j0, ws.g_used, adv, ell_old, loss_scale, ell, g, loss,
                                        flags, ws.seq_scale, ws.row_scale, backward ? 1 : 0, bound,
                                        dbar);
  return hipGetLastError();
}

// dbar[b] = (1/n_t) sum_j (l[b][j] - l_old[b][j]), samples in order: the
// log-ratio B_theta - B_old of Eq. elbo_ratio with both ELBOs estimated on the
// same n_t masked samples.
__global__ __launch_bounds__(256) void k_mean_ratio(const double* __restrict__ ell,
                                                    const double* __restrict__ ell_old, int B,
                                                    int n_t, double* __restrict__ dbar) {
  const int b = blockIdx.x * 256 + threadIdx.x;
  if (b >= B) return;
  double acc = 0.0;
  for (int j = 0; j < n_t; ++j) acc += ell[(int64_t)b * n_t + j] - ell_old[(int64_t)b * n_t + j];
  dbar[b] = acc / n_t;
}

hipError_t launch_mean_ratio(const double* ell, const double* ell_old, int B, int n_t,
                             double* dbar, hipStream_t s) {
  k_mean_ratio<<<(unsigned)((B + 255) / 256), 256, 0, s>>>(ell, ell_old, B, n_t, dbar);
  return hipGetLastError();
}

// Stored backward, once the unit's scales s are known.  The forward kept
// u = 2^(z log2e - R2) (bf16) in dZ (the unit's rows from its col_off, ldz
// rows per slab), with R2 = exp_reference(z_y)
// per row; since p = u 2^(R2 - lse2),
//     dZ = s (p - onehot) = f (u - onehot 2^(lse2 - R2)),  f = s 2^(R2 - lse2)
// (differentiating Eq. per_step_loss, d l / d z = (onehot - p) / t; s carries
// -loss_scale dg/dl and the 1/t).  k_grad_rows sets f per row (0 for padding)
// and replaces the target entry by (p_y - 1) 2^(lse2 - R2),
// p_y from the fp32 target logit; f scales the dX rows in the reduction and
// H_c^T's columns (k_scale_hct) for the dW GEMM.  A row with
// lse2 - R2 > kExpRange (its target log2-probability below
// -(kExpRef + kExpRange)) is marked: its exponentials may have left the range
// of bf16 and of the fp32 accumulators, so k_fixup_rows recomputes the row
// against R2 = lse2 (f = s), from fp32 dot products.
__global__ __launch_bounds__(256) void k_grad_rows(
    const float* __restrict__ lse2, const float* __restrict__ row_scale,
    const float* __restrict__ ztgt, const int32_t* __restrict__ row_tgt,
    const SampleMeta* __restrict__ meta, uint16_t* __restrict__ dZ, float* __restrict__ row_f,
    uint8_t* __restrict__ row_bad, int64_t ldz) {
  const int r = blockIdx.x * 256 + threadIdx.x;
  if (r >= meta->n_rows_pad) return;
  float f = 0.f;
  if (r < meta->n_rows) {
    const float l2 = lse2[r], z2 = ztgt[r] * kLog2e;
    const float r2 = exp_reference(ztgt[r]);
    const bool bad = !(l2 - r2 <= kExpRange);   // (NaN too)
    const float r2e = bad ? l2 : r2;
    f = row_scale[r] * __builtin_amdgcn_exp2f(r2e - l2);
    const float val = (__builtin_amdgcn_exp2f(z2 - l2) - 1.f) * __builtin_amdgcn_exp2f(l2 - r2e);
    const uint16_t b = (uint16_t)(pack_bf16x2(val, 0.f) & 0xFFFFu);
    const int y = row_tgt[r];
    dZ[slab_index(ldz, (int64_t)meta->col_off + r, y)] = b;
    row_bad[r] = bad;
  }
  row_f[r] = f;
}

// H_c^T[c][col_off + r] *= f_r (bf16, nearest even) over the unit's columns
// up to col_end (its rows rounded up to 64), not its 256-row padding: the next
// unit of the dW batch starts at col_end, and with every sample retained its
// columns already hold its rows when this runs.  One workgroup per 64 x 64
// tile, which is 8 KB of the slab-major H_c^T.
__global__ __launch_bounds__(256) void k_scale_hct(const float* __restrict__ row_f,
                                                   const SampleMeta* __restrict__ meta,
                                                   uint16_t* __restrict__ HcT, int d) {
  const int r0 = blockIdx.x * 64, c0 = blockIdx.y * 64;
  if (r0 >= meta->col_end - meta->col_off) return;
  const int tid = threadIdx.x, cc = tid & 7;
  float fr[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) fr[e] = row_f[r0 + cc * 8 + e];
  uint16_t* base = HcT + slab_index(d, c0, (int64_t)meta->col_off + r0);
#pragma unroll
  for (int it = 0; it < 2; ++it) {
    const int c = (tid >> 3) + 32 * it;
    uint4* q = reinterpret_cast<uint4*>(base + (int64_t)c * 64 + cc * 8);
    const uint4 v = *q;
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
    uint32_t o[4];
#pragma unroll
    for (int e = 0; e < 4; ++e)
      o[e] = pack_bf16x2(__uint_as_float(w[e] << 16) * fr[2 * e],
                         __uint_as_float(w[e] & 0xFFFF0000u) * fr[2 * e + 1]);
    *q = make_uint4(o[0], o[1], o[2], o[3]);
  }
}

// The marked rows of the unit, recomputed against R2 = lse2:
// u = 2^(z log2e - lse2) = p, and p_y - 1 at the target.  One
// thread per vocabulary id; each workgroup scans the unit's marks 256 rows at
// a time and takes the marked ones in batches of 16, whose fp32 logits
// z = H_c[row] . W^T[v] it accumulates in a fixed order over d.  Without
// marked rows it only reads the marks.
constexpr int kFixBatch = 16;

__global__ __launch_bounds__(256) void k_fixup_rows(
    const uint16_t* __restrict__ Hc, const uint16_t* __restrict__ WT,
    const float* __restrict__ lse2, const float* __restrict__ ztgt,
    const int32_t* __restrict__ row_tgt, const uint8_t* __restrict__ row_bad,
    const SampleMeta* __restrict__ meta, uint16_t* __restrict__ dZ, int d, int V, int64_t RP,
    int64_t ldz) {
  __shared__ int s_list[256];
  __shared__ int s_cnt;
  __shared__ float s_h[kFixBatch][64];
  const int tid = threadIdx.x;
  const int v = blockIdx.x * 256 + tid;
  const int N = meta->n_rows;
  const int64_t col_off = meta->col_off;
  for (int base = 0; base < N; base += 256) {
    if (tid == 0) s_cnt = 0;
    __syncthreads();
    const int rr = base + tid;
    if (rr < N && row_bad[rr]) s_list[atomicAdd(&s_cnt, 1)] = rr;
    __syncthreads();
    const int cnt = s_cnt;
    for (int b0 = 0; b0 < cnt; b0 += kFixBatch) {
      const int nb = min(kFixBatch, cnt - b0);
      float acc[kFixBatch];
#pragma unroll
      for (int i = 0; i < kFixBatch; ++i) acc[i] = 0.f;
      for (int kc = 0; kc < d; kc += 64) {
        __syncthreads();
        for (int q = tid; q < kFixBatch * 64; q += 256) {
          const int i = q >> 6, k = q & 63;
          s_h[i][k] = i < nb ? __uint_as_float((uint32_t)Hc[slab_index(RP, s_list[b0 + i], kc + k)] << 16)
                             : 0.f;
        }
        __syncthreads();
        if (v < V) {
          const uint16_t* w = WT + (int64_t)v * d + kc;
          for (int kk = 0; kk < 64; kk += 8) {
            const uint4 wv = *reinterpret_cast<const uint4*>(w + kk);
            const uint32_t ww[4] = {wv.x, wv.y, wv.z, wv.w};
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              const float w0 = __uint_as_float(ww[e] << 16), w1 = __uint_as_float(ww[e] & 0xFFFF0000u);
#pragma unroll
              for (int i = 0; i < kFixBatch; ++i)
                acc[i] = fmaf(w1, s_h[i][kk + 2 * e + 1], fmaf(w0, s_h[i][kk + 2 * e], acc[i]));
            }
          }
        }
      }
      if (v < V) {
#pragma unroll
        for (int i = 0; i < kFixBatch; ++i) {
          if (i >= nb) break;
          const int r = s_list[b0 + i];
          const float l2 = lse2[r];
          const float val = v == row_tgt[r] ? __builtin_amdgcn_exp2f(fmaf(ztgt[r], kLog2e, -l2)) - 1.f
                                            : __builtin_amdgcn_exp2f(fmaf(acc[i], kLog2e, -l2));
          const uint16_t b = (uint16_t)(pack_bf16x2(val, 0.f) & 0xFFFFu);
          dZ[slab_index(ldz, col_off + r, v)] = b;
        }
      }
    }
    __syncthreads();   // s_list / s_cnt are rewritten for the next rows
  }
}

hipError_t launch_grad_scale(const Workspace& ws, int d, int V, hipStream_t s) {
  k_grad_rows<<<(unsigned)(ws.RP / 256), 256, 0, s>>>(ws.lse2, ws.row_scale, ws.ztgt, ws.row_tgt,
                                                      ws.unit(), ws.dZ, ws.row_f, ws.row_bad,
                                                      ws.ldz);
  if (hipError_t e = hipGetLastError(); e != hipSuccess) return e;
  k_scale_hct<<<dim3((unsigned)(ws.RP / 64), (unsigned)(d / 64)), 256, 0, s>>>(ws.row_f, ws.unit(),
                                                                             ws.HcT, d);
  if (hipError_t e = hipGetLastError(); e != hipSuccess) return e;
  k_fixup_rows<<<(unsigned)((V + 255) / 256), 256, 0, s>>>(ws.Hc, ws.WT, ws.lse2, ws.ztgt,
                                                           ws.row_tgt, ws.row_bad, ws.unit(),
                                                           ws.dZ, d, V, ws.RP, ws.ldz);
  return hipGetLastError();
}

// dX[idx[r], :] += f_r sum_s part[s][r][:] over the rows r of one sample of
// the unit (sm: its record; um: the unit's, which holds the split count; f_r
// the stored backward's row factor, 1 without one), float4 per thread; rows
// are unique within a sample, so there are no write conflicts.
__global__ __launch_bounds__(256) void k_dx_reduce(const float* __restrict__ part,
                                                   const int32_t* __restrict__ idx,
                                                   const SampleMeta* __restrict__ sm,
                                                   const SampleMeta* __restrict__ um,
                                                   const float* __restrict__ rowf,
                                                   float* __restrict__ dX, int d,
                                                   int64_t split_stride) {
  if ((int)blockIdx.x >= sm->s_rows) return;
  const int r = sm->s_row_off + blockIdx.x;
  const int n_split = um->dx_split;
  const int c = (blockIdx.y * 256 + threadIdx.x) * 4;
  if (c >= d) return;
  float4 acc = *reinterpret_cast<const float4*>(part + (int64_t)r * d + c);
  for (int s = 1; s < n_split; ++s) {
    const float4 v = *reinterpret_cast<const float4*>(part + s * split_stride + (int64_t)r * d + c);
    acc.x += v.x; acc.y += v.y; acc.z += v.z; acc.w += v.w;
  }
  if (rowf) {
    const float f = rowf[r];
    acc.x *= f; acc.y *= f; acc.z *= f; acc.w *= f;
  }
  float4* dst = reinterpret_cast<float4*>(dX + (int64_t)idx[r] * d + c);
  float4 o = *dst;
  o.x += acc.x; o.y += acc.y; o.z += acc.z; o.w += acc.w;
  *dst = o;
}

hipError_t launch_dx_reduce(const Workspace& ws, int g, float* dX, int d, hipStream_t s) {
  dim3 grid((unsigned)ws.NP, (unsigned)((d / 4 + 255) / 256));
  k_dx_reduce<<<grid, 256, 0, s>>>(ws.dx_part, ws.idx, ws.meta + g, ws.unit(),
                                   ws.chunk ? nullptr : ws.row_f, dX, d, ws.RP * d);
  return hipGetLastError();
}

// Split reduction followed by the backward of the final RMSNorm
// h = gamma x r, r = (mean x^2 + eps)^(-1/2), for one row of one sample of the
// unit per workgroup (x: that sample's activations):
//   dh       = f_row sum_s part[s][row]               (d loss / d h; f_row the
//                                                     stored backward's row
//                                                     factor, 1 without one)
//   dx_k    += r gamma_k dh_k - (r^3 / d) x_k sum_i gamma_i dh_i x_i
//   c_k      = dh_k x_k r  -> part[0][row][k], summed over rows into dgamma
// Every thread revisits only the elements it wrote, so part[0] needs no
// cross-thread ordering; the row dot product goes through LDS.
template <typename T>
__global__ __launch_bounds__(256) void k_dx_reduce_rmsnorm(
    float* __restrict__ part, const int32_t* __restrict__ idx, const SampleMeta* __restrict__ sm,
    const SampleMeta* __restrict__ um, const float* __restrict__ rowf, const T* __restrict__ x,
    const float* __restrict__ gamma, const float* __restrict__ inv_rms, float* __restrict__ dx,
    int d, int64_t split_stride) {
  __shared__ float red[4];
  if ((int)blockIdx.x >= sm->s_rows) return;
  const int r = sm->s_row_off + blockIdx.x;
  const int n_split = um->dx_split;
  const int tid = threadIdx.x;
  const float f = rowf ? rowf[r] : 1.f;   // the stored backward's row factor
  float* p0 = part + (int64_t)r * d;
  const T* xr = x + (int64_t)idx[r] * d;
  float dot = 0.f;
  for (int c = tid * 4; c < d; c += 1024) {
    float4 acc = *reinterpret_cast<const float4*>(p0 + c);
    for (int sp = 1; sp < n_split; ++sp) {
      const float4 v = *reinterpret_cast<const float4*>(p0 + sp * split_stride + c);
      acc.x += v.x; acc.y += v.y; acc.z += v.z; acc.w += v.w;
    }
    acc.x *= f; acc.y *= f; acc.z *= f; acc.w *= f;
    *reinterpret_cast<float4*>(p0 + c) = acc;
    const uint2 xv = load_bf16x4(xr + c);
    const float4 g = *reinterpret_cast<const float4*>(gamma + c);
    dot = fmaf(g.x * acc.x, __uint_as_float(xv.x << 16), dot);
    dot = fmaf(g.y * acc.y, __uint_as_float(xv.x & 0xFFFF0000u), dot);
    dot = fmaf(g.z * acc.z, __uint_as_float(xv.y << 16), dot);
    dot = fmaf(g.w * acc.w, __uint_as_float(xv.y & 0xFFFF0000u), dot);
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) dot += __shfl_xor(dot, off, 64);
  if ((tid & 63) == 0) red[tid >> 6] = dot;
  __syncthreads();
  dot = red[0] + red[1] + red[2] + red[3];
  const float ir = inv_rms[r];
  const float cx = ir * ir * ir * dot / (float)d;
  float* dxr = dx + (int64_t)idx[r] * d;
  for (int c = tid * 4; c < d; c += 1024) {
    const float4 dh = *reinterpret_cast<const float4*>(p0 + c);
    const uint2 xv = load_bf16x4(xr + c);
    const float4 g = *reinterpret_cast<const float4*>(gamma + c);
    const float x0 = __uint_as_float(xv.x << 16), x1 = __uint_as_float(xv.x & 0xFFFF0000u);
    const float x2 = __uint_as_float(xv.y << 16), x3 = __uint_as_float(xv.y & 0xFFFF0000u);
    float4 o = *reinterpret_cast<float4*>(dxr + c);
    o.x += ir * g.x * dh.x - cx * x0;
    o.y += ir * g.y * dh.y - cx * x1;
    o.z += ir * g.z * dh.z - cx * x2;
    o.w += ir * g.w * dh.w - cx * x3;
    *reinterpret_cast<float4*>(dxr + c) = o;
    *reinterpret_cast<float4*>(p0 + c) = make_float4(dh.x * x0 * ir, dh.y * x1 * ir, dh.z * x2 * ir, dh.w * x3 * ir);
  }
}

// dgamma[k] += sum over one sample's rows of part[0][row][k], in a fixed
// order: partial sums over 256-row chunks of the sample, then the chunks in
// order.
__global__ __launch_bounds__(256) void k_dgamma_partial(const float* __restrict__ part,
                                                        const SampleMeta* __restrict__ sm,
                                                        float* __restrict__ gpart, int d) {
  const int k = blockIdx.x * 256 + threadIdx.x;
  const int r0 = blockIdx.y * 256;
  if (k >= d) return;
  const int r1 = min(sm->s_rows, r0 + 256);
  const float* base = part + (int64_t)sm->s_row_off * d;
  float acc = 0.f;
  for (int r = r0; r < r1; ++r) acc += base[(int64_t)r * d + k];
  gpart[(int64_t)blockIdx.y * d + k] = acc;
}

__global__ __launch_bounds__(256) void k_dgamma_final(const float* __restrict__ gpart,
                                                      const SampleMeta* __restrict__ sm,
                                                      float* __restrict__ dgamma, int d) {
  const int k = blockIdx.x * 256 + threadIdx.x;
  if (k >= d) return;
  const int chunks = (sm->s_rows + 255) / 256;
  float acc = 0.f;
  for (int c = 0; c < chunks; ++c) acc += gpart[(int64_t)c * d + k];
  dgamma[k] += acc;
}

hipError_t launch_dx_reduce_rmsnorm(const Workspace& ws, int g, const void* x, bool f32,
                                    const float* gamma, float* dx, float* dgamma, int d,
                                    hipStream_t s) {
  const SampleMeta* sm = ws.meta + g;
  if (f32)
    k_dx_reduce_rmsnorm<float><<<(unsigned)ws.NP, 256, 0, s>>>(
        ws.dx_part, ws.idx, sm, ws.unit(), ws.chunk ? nullptr : ws.row_f,
        static_cast<const float*>(x), gamma, ws.inv_rms, dx, d, ws.RP * d);
  else
    k_dx_reduce_rmsnorm<uint16_t><<<(unsigned)ws.NP, 256, 0, s>>>(
        ws.dx_part, ws.idx, sm, ws.unit(), ws.chunk ? nullptr : ws.row_f,
        static_cast<const uint16_t*>(x), gamma, ws.inv_rms, dx, d, ws.RP * d);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  dim3 g1((unsigned)((d + 255) / 256), (unsigned)(ws.NP / 256));
  k_dgamma_partial<<<g1, 256, 0, s>>>(ws.dx_part, sm, ws.gpart, d);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  k_dgamma_final<<<(unsigned)((d + 255) / 256), 256, 0, s>>>(ws.gpart, sm, dgamma, d);
  return hipGetLastError();
}

}  // namespace bgpo
