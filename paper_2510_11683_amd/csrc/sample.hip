// Timestep draw, Bernoulli(t) masking, stable stream compaction of the masked
// positions, gather of the masked hidden rows, and the one-off W_head
// transpose.
//
// The forward masking process (Section 2.1) masks every response token
// independently with probability t; the ELBO term (Eq. per_step_loss) only
// touches masked positions, so the rows that reach the LM-head GEMMs are the
// masked ones, compacted in ascending flat order b*L + i.
#include "common.hpp"
#include "internal.hpp"

namespace bgpo {

constexpr int kMaskThreads = 1024;
constexpr int kMaxB = 4096;
// the single-workgroup mask kernel takes problems up to this many positions;
// larger ones go through the multi-block passes below
constexpr int64_t kSingleBlockPositions = 65536;

// Philox words for position p = b*L + i are taken from counter (i>>2, seq, j, 0);
// consecutive positions of one response share a counter block, so a thread
// caches the last block it computed.
struct MaskWalker {
  uint32_t k0, k1, seq_base;
  int L, j;
  int cached_b = -1, cached_blk = -1;
  u32x4 w;
  __device__ bool masked(const uint8_t* resp, const uint32_t* sT, int64_t p) {
    return resp[p] ? test(sT, p) : false;
  }
  // the Philox test of response position p (resp_mask[p] != 0 assumed)
  __device__ bool test(const uint32_t* sT, int64_t p) {
    const int b = (int)(p / L);
    const int i = (int)(p - (int64_t)b * L);
    const int blk = i >> 2;
    if (blk != cached_blk || b != cached_b) {
      w = philox4x32_10(u32x4{(uint32_t)blk, seq_base + (uint32_t)b, (uint32_t)j, 0u}, k0, k1);
      cached_blk = blk;
      cached_b = b;
    }
    return (pick_word(w, i & 3) >> 8) < sT[b];
  }
};

// Vocabulary split of the dX GEMM for a unit with row_tiles 256-row tiles:
// the split count s minimising an estimate of the GEMM's time on the
// persistent grid, in units of one 256x256x64 slab on one workgroup:
//   ceil(tiles / grid) rounds x (slabs per split + ~10 for the tile's
//   prologue and fp32 partial store) + ~0.65 per (split, row tile) for the
//   reduction of the partials.
// A fixed split leaves most of the last round idle for some row counts
// (576 tiles on 256 workgroups use 2.25 of 3 rounds).
__device__ void choose_dx_split(int row_tiles, const DxPlan& pl, int* split, int* kslab) {
  // 32-bit divisions (tiles <= 16384 x 256 x 16), 64-bit cost
  int best_s = 1, best_ks = pl.kslabs;
  uint64_t best = ~0ull;
  for (int sp = 1; sp <= pl.s_max && row_tiles > 0; ++sp) {
    const uint32_t ks = ((uint32_t)pl.kslabs + sp - 1) / sp;
    const uint32_t se = ((uint32_t)pl.kslabs + ks - 1) / ks;   // splits actually used
    const uint32_t tiles = (uint32_t)row_tiles * pl.col_tiles * se;
    const uint32_t rounds = (tiles + pl.grid - 1) / pl.grid;
    const uint64_t cost = (uint64_t)rounds * (ks + 10) * 20 + 13ull * se * row_tiles;
    if (cost < best) {
      best = cost;
      best_s = (int)se;
      best_ks = (int)ks;
    }
  }
  *split = best_s;
  *kslab = best_ks;
}

// Pointers of a unit's row state handed to the mask kernel (all NULL for the
// mask-only test hook, which writes positions to idx at row 0).
struct MaskOut {
  int32_t* idx;          // [rows]  masked flat positions, indexed by unit row
  int32_t* row_tgt;      // [rows]  target token
  int32_t* row_seq;      // [rows]  g*B + b
  int32_t* seg_off;      // [B+1]   this sample's response offsets (unit rows)
  uint32_t* t24;         // [B]     this sample's timesteps
  SampleMeta* meta;      // this sample's record
  int row_cap;           // rows the unit holds (padding is written up to it)
};

// The record of a sample whose `total` masked rows follow row0 rows of its
// unit, with the unit's columns from col0.
__device__ void write_record(SampleMeta* m, int row0, int col0, int total, const DxPlan& plan) {
  if (!m) return;
  const int rows = row0 + total;
  const int rows_pad = (rows + kRowPad - 1) / kRowPad * kRowPad;
  m->n_rows = rows;
  m->n_rows_pad = rows_pad;
  m->col_off = col0;
  m->col_end = col0 + (rows + 63) / 64 * 64;
  m->s_rows = total;
  m->s_row_off = row0;
  choose_dx_split(rows_pad / kRowPad, plan, &m->dx_split, &m->dx_kslab);
}

// Single-workgroup form (up to kSingleBlockPositions positions): timesteps in
// LDS, every thread a contiguous run of positions, one block-wide scan.
__global__ __launch_bounds__(kMaskThreads) void k_mask_compact(
    const uint8_t* __restrict__ resp, const int32_t* __restrict__ targets, int B, int L, int n_t,
    int j, int g, int t_mode, uint32_t k0, uint32_t k1, uint32_t seq_base, MaskOut out,
    int32_t* __restrict__ nm_out, int nm_stride, float* __restrict__ t_out, int t_stride, int V,
    const SampleMeta* prev, DxPlan plan) {
  __shared__ uint32_t sT[kMaxB];
  __shared__ int32_t sSeg[kMaxB + 1];
  __shared__ int32_t sWave[kMaskThreads / 64];
  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;

  // where this sample's rows start: after the unit's earlier samples (g > 0),
  // or at row 0 of a new unit whose columns follow the previous unit's
  const int row0 = (g > 0 && prev) ? prev->n_rows : 0;
  const int col0 = prev ? (g > 0 ? prev->col_off : prev->col_end) : 0;

  for (int b = tid; b < B; b += kMaskThreads)
    sT[b] = timestep_t24(k0, k1, seq_base + (uint32_t)b, j, n_t, t_mode);
  __syncthreads();

  const int64_t P = (int64_t)B * L;
  const int64_t chunk = (P + kMaskThreads - 1) / kMaskThreads;
  const int64_t p0 = min(P, (int64_t)tid * chunk), p1 = min(P, p0 + chunk);

  MaskWalker mw{k0, k1, seq_base, L, j};
  int cnt = 0;
  for (int64_t p = p0; p < p1; ++p) cnt += mw.masked(resp, sT, p) ? 1 : 0;

  // block-wide exclusive scan of the per-thread counts
  int incl = cnt;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const int v = __shfl_up(incl, off, 64);
    if (lane >= off) incl += v;
  }
  if (lane == 63) sWave[wave] = incl;
  __syncthreads();
  if (wave == 0) {
    int wv = lane < kMaskThreads / 64 ? sWave[lane] : 0;
    int wincl = wv;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const int v = __shfl_up(wincl, off, 64);
      if (lane >= off) wincl += v;
    }
    if (lane < kMaskThreads / 64) sWave[lane] = wincl - wv;  // exclusive
  }
  __syncthreads();
  int base = sWave[wave] + incl - cnt;

  MaskWalker mw2{k0, k1, seq_base, L, j};
  for (int64_t p = p0; p < p1; ++p) {
    const int b = (int)(p / L);
    if (p == (int64_t)b * L) sSeg[b] = base;
    if (mw2.masked(resp, sT, p)) {
      const int r = row0 + base;
      if (out.idx) out.idx[r] = (int32_t)p;
      if (out.row_tgt) {
        // ids outside [0, V) are clamped so that no kernel reads outside W
        const int y = targets[p];
        out.row_tgt[r] = y < 0 ? 0 : (y >= V ? V - 1 : y);
      }
      if (out.row_seq) out.row_seq[r] = g * B + b;
      ++base;
    }
  }
  if (tid == kMaskThreads - 1) sSeg[B] = base;  // the last thread ends at P
  __syncthreads();

  const int total = sSeg[B];
  const int rows = row0 + total;
  const int rows_pad = (rows + kRowPad - 1) / kRowPad * kRowPad;
  for (int b = tid; b < B; b += kMaskThreads) {
    const int nm = sSeg[b + 1] - sSeg[b];
    if (nm_out) nm_out[(int64_t)b * nm_stride] = nm;
    if (t_out) t_out[(int64_t)b * t_stride] = (float)sT[b] * (1.0f / 16777216.0f);
    if (out.seg_off) out.seg_off[b] = row0 + sSeg[b];
    if (out.t24) out.t24[b] = sT[b];
  }
  if (tid == 0) {
    if (out.seg_off) out.seg_off[B] = rows;
    write_record(out.meta, row0, col0, total, plan);
  }
  // padding rows up to the next row tile (a later sample of the unit
  // overwrites them with its own rows)
  const int pad_end = min(rows_pad, out.row_cap);
  for (int r = rows + tid; r < pad_end; r += kMaskThreads) {
    if (out.row_tgt) out.row_tgt[r] = 0;
    if (out.row_seq) out.row_seq[r] = 0;
  }
}

// ---------------------------------------------------------------------------
// Multi-block form for large B*L: the same masks (the same Philox words and
// integer test), in three passes that each spread over the whole GPU:
//   k_mask_bits     one 32-bit mask word per thread (32 consecutive positions),
//                   one count per block of kMbPositions positions
//   k_mask_scan     one block: exclusive scan of the block counts, the
//                   per-response offsets (block offset + popcounts of the
//                   words before the response's first position), counts,
//                   the sample's record and the padding rows
//   k_mask_scatter  every set bit in ascending position order to its row
// so the compacted order and every count equal the single-block form's.
constexpr int kMbThreads = 256;
constexpr int kMbPositions = kMbThreads * 32;   // positions per block

__global__ __launch_bounds__(256) void k_timesteps(int B, int n_t, int j, int t_mode, uint32_t k0,
                                                   uint32_t k1, uint32_t seq_base,
                                                   uint32_t* __restrict__ t24,
                                                   float* __restrict__ t_out, int t_stride) {
  const int b = blockIdx.x * 256 + threadIdx.x;
  if (b >= B) return;
  const uint32_t T = timestep_t24(k0, k1, seq_base + (uint32_t)b, j, n_t, t_mode);
  t24[b] = T;
  if (t_out) t_out[(int64_t)b * t_stride] = (float)T * (1.0f / 16777216.0f);
}

// exclusive prefix of v over the block's 256 threads (and the block total)
__device__ __forceinline__ int block_exclusive_sum(int v, int* s_wave, int* total) {
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  int incl = v;
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    const int u = __shfl_up(incl, off, 64);
    if (lane >= off) incl += u;
  }
  if (lane == 63) s_wave[wave] = incl;
  __syncthreads();
  int base = incl - v;
  for (int q = 0; q < wave; ++q) base += s_wave[q];
  *total = s_wave[0] + s_wave[1] + s_wave[2] + s_wave[3];
  return base;
}

__global__ __launch_bounds__(kMbThreads) void k_mask_bits(
    const uint8_t* __restrict__ resp, const uint32_t* __restrict__ t24, int L, int64_t P, int j,
    uint32_t k0, uint32_t k1, uint32_t seq_base, uint32_t* __restrict__ bits,
    int32_t* __restrict__ wprefix, int32_t* __restrict__ blk_count) {
  __shared__ int s_wave[kMbThreads / 64];
  const int tid = threadIdx.x;
  const int64_t w = (int64_t)blockIdx.x * kMbThreads + tid;
  uint32_t word = 0;
  const int64_t p0 = w * 32;
  if (p0 < P) {
    // the word's 32 response-mask bytes in two 16-byte loads (resp_mask rows
    // are contiguous; a word that crosses P reads byte by byte)
    uint8_t r[32];
    if (p0 + 32 <= P && (((uintptr_t)(resp + p0)) & 15) == 0) {
      *reinterpret_cast<uint4*>(r) = *reinterpret_cast<const uint4*>(resp + p0);
      *reinterpret_cast<uint4*>(r + 16) = *reinterpret_cast<const uint4*>(resp + p0 + 16);
    } else {
#pragma unroll
      for (int e = 0; e < 32; ++e) r[e] = p0 + e < P ? resp[p0 + e] : 0;
    }
    MaskWalker mw{k0, k1, seq_base, L, j};
#pragma unroll
    for (int e = 0; e < 32; ++e)
      if (r[e] && mw.test(t24, p0 + e)) word |= 1u << e;
    bits[w] = word;
  }
  int total;
  const int pre = block_exclusive_sum(__popc(word), s_wave, &total);
  if (p0 < P) wprefix[w] = pre;
  if (tid == 0) blk_count[blockIdx.x] = total;
}

constexpr int kMbMaxBlocks = (1 << 20) / kMbPositions;   // B*L <= 2^20

// masked positions before position pos < P: the block's offset, the word's
// prefix within its block, the word's bits below pos
__device__ __forceinline__ int masked_before(const uint32_t* bits, const int32_t* wprefix,
                                             const int32_t* blk_off, int64_t pos) {
  const int64_t w = pos / 32;
  return blk_off[w / kMbThreads] + wprefix[w] +
         __popc(bits[w] & ((1u << (int)(pos - w * 32)) - 1u));
}

__global__ __launch_bounds__(1024) void k_mask_scan(
    const uint32_t* __restrict__ bits, const int32_t* __restrict__ wprefix,
    const int32_t* __restrict__ blk_count,
    int32_t* __restrict__ blk_off, int nblk, int B, int L, int g, MaskOut out,
    int32_t* __restrict__ nm_out, int nm_stride, const SampleMeta* prev, DxPlan plan) {
  __shared__ int s_total;
  __shared__ int32_t s_off[kMbMaxBlocks];
  const int tid = threadIdx.x;
  if (tid == 0) {
    int acc = 0;
    for (int q = 0; q < nblk; ++q) {
      s_off[q] = acc;
      blk_off[q] = acc;   // for the scatter pass
      acc += blk_count[q];
    }
    s_total = acc;
  }
  __syncthreads();
  const int total = s_total;
  const int row0 = (g > 0 && prev) ? prev->n_rows : 0;
  const int col0 = prev ? (g > 0 ? prev->col_off : prev->col_end) : 0;
  for (int b = tid; b < B; b += 1024) {
    const int s0 = masked_before(bits, wprefix, s_off, (int64_t)b * L);
    const int s1 = b + 1 < B ? masked_before(bits, wprefix, s_off, (int64_t)(b + 1) * L) : total;
    if (nm_out) nm_out[(int64_t)b * nm_stride] = s1 - s0;
    if (out.seg_off) out.seg_off[b] = row0 + s0;
  }
  const int rows = row0 + total;
  const int rows_pad = (rows + kRowPad - 1) / kRowPad * kRowPad;
  if (tid == 0) {
    if (out.seg_off) out.seg_off[B] = rows;
    write_record(out.meta, row0, col0, total, plan);
  }
  const int pad_end = min(rows_pad, out.row_cap);
  for (int r = rows + tid; r < pad_end; r += 1024) {
    if (out.row_tgt) out.row_tgt[r] = 0;
    if (out.row_seq) out.row_seq[r] = 0;
  }
}

__global__ __launch_bounds__(kMbThreads) void k_mask_scatter(
    const uint32_t* __restrict__ bits, const int32_t* __restrict__ wprefix,
    const int32_t* __restrict__ blk_off, const int32_t* __restrict__ targets, int B, int L,
    int64_t P, int g, int V, MaskOut out, const SampleMeta* prev) {
  const int64_t w = (int64_t)blockIdx.x * kMbThreads + threadIdx.x;
  if (w * 32 >= P) return;
  const uint32_t word = bits[w];
  const int row0 = (g > 0 && prev) ? prev->n_rows : 0;
  int r = row0 + blk_off[blockIdx.x] + wprefix[w];
  uint32_t m = word;
  while (m) {
    const int e = __builtin_ctz(m);
    m &= m - 1;
    const int64_t p = w * 32 + e;
    if (out.idx) out.idx[r] = (int32_t)p;
    if (out.row_tgt) {
      const int y = targets[p];
      out.row_tgt[r] = y < 0 ? 0 : (y >= V ? V - 1 : y);
    }
    if (out.row_seq) out.row_seq[r] = g * B + (int)(p / L);
    ++r;
  }
}

size_t mask_scratch_bytes(int B, int L) {
  const int64_t P = (int64_t)B * L;
  const int64_t words = (P + 31) / 32, nblk = (P + kMbPositions - 1) / kMbPositions;
  return (size_t)(words * 8 + nblk * 8 + (int64_t)B * 4 + 4 * 256);
}

hipError_t launch_mask_compact(const uint8_t* resp, const int32_t* targets, int B, int L, int n_t,
                               int j, int g, int t_mode, uint64_t seed, uint32_t seq_base,
                               const Workspace* ws, int32_t* idx_out, int32_t* n_masked_out,
                               int nm_stride, float* t_out, int t_stride, int V,
                               const SampleMeta* prev, const DxPlan& plan, void* scratch,
                               bool force_multi, hipStream_t s) {
  MaskOut out{idx_out, nullptr, nullptr, nullptr, nullptr, nullptr, 0};
  if (ws) {
    out.idx = ws->idx;
    out.row_tgt = ws->row_tgt;
    out.row_seq = ws->row_seq;
    out.seg_off = ws->seg_off + (int64_t)g * (B + 1);
    out.t24 = ws->t24 + (int64_t)g * B;
    out.meta = ws->meta + g;
    out.row_cap = (int)ws->RP;
  }
  const uint32_t k0 = (uint32_t)(seed & 0xFFFFFFFFu), k1 = (uint32_t)(seed >> 32);
  const int64_t P = (int64_t)B * L;
  if ((P <= kSingleBlockPositions && !force_multi) || !scratch) {
    k_mask_compact<<<1, kMaskThreads, 0, s>>>(resp, targets, B, L, n_t, j, g, t_mode, k0, k1,
                                              seq_base, out, n_masked_out, nm_stride, t_out,
                                              t_stride, V, prev, plan);
    return hipGetLastError();
  }
  // scratch: mask words, block counts and offsets, and (without a unit) the
  // sample's timesteps
  char* sc = static_cast<char*>(scratch);
  const int64_t words = (P + 31) / 32, nblk = (P + kMbPositions - 1) / kMbPositions;
  const int64_t wbytes = (words * 4 + 255) / 256 * 256;
  uint32_t* bits = reinterpret_cast<uint32_t*>(sc);
  int32_t* wprefix = reinterpret_cast<int32_t*>(sc + wbytes);
  int32_t* blk_count = reinterpret_cast<int32_t*>(sc + 2 * wbytes);
  int32_t* blk_off = blk_count + nblk;
  uint32_t* t24 = out.t24 ? out.t24
                          : reinterpret_cast<uint32_t*>(sc + 2 * wbytes +
                                                        (nblk * 8 + 255) / 256 * 256);
  k_timesteps<<<(unsigned)((B + 255) / 256), 256, 0, s>>>(B, n_t, j, t_mode, k0, k1, seq_base, t24,
                                                          t_out, t_stride);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  k_mask_bits<<<(unsigned)nblk, kMbThreads, 0, s>>>(resp, t24, L, P, j, k0, k1, seq_base, bits,
                                                    wprefix, blk_count);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  k_mask_scan<<<1, 1024, 0, s>>>(bits, wprefix, blk_count, blk_off, (int)nblk, B, L, g, out,
                                 n_masked_out, nm_stride, prev, plan);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  k_mask_scatter<<<(unsigned)nblk, kMbThreads, 0, s>>>(bits, wprefix, blk_off, targets, B, L, P,
                                                       g, V, out, prev);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Inverse RMS of the masked rows of the pre-norm activations x (for the final
// RMSNorm h = gamma x r, r = (mean x^2 + eps)^(-1/2)): one wave per row, fp32
// sum of squares.  Row r of the unit reads sample g = row_seq[r] / B, i.e.
// x + g * stride.
template <typename T>
__global__ __launch_bounds__(256) void k_row_rms(const T* __restrict__ x, int64_t stride,
                                                 int B, const int32_t* __restrict__ idx,
                                                 const int32_t* __restrict__ row_seq,
                                                 const SampleMeta* __restrict__ meta,
                                                 float* __restrict__ inv_rms, int d, float eps) {
  const int row = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (row >= meta->n_rows) return;
  const T* xr = x + (int64_t)(row_seq[row] / B) * stride + (int64_t)idx[row] * d;
  float acc = 0.f;
  for (int k = lane * 8; k < d; k += 64 * 8) {
    const uint4 v = load_bf16x8(xr + k);
    const uint32_t a[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const float lo = __uint_as_float(a[e] << 16), hi = __uint_as_float(a[e] & 0xFFFF0000u);
      acc = fmaf(lo, lo, acc);
      acc = fmaf(hi, hi, acc);
    }
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) acc += __shfl_xor(acc, off, 64);
  if (lane == 0) inv_rms[row] = 1.f / sqrtf(acc / (float)d + eps);
}

hipError_t launch_row_rms(const void* x, bool f32, int64_t stride, int B, const Workspace& ws,
                          int d, float eps, hipStream_t s) {
  const unsigned grid = (unsigned)(ws.RP / 4);
  if (f32)
    k_row_rms<float><<<grid, 256, 0, s>>>(static_cast<const float*>(x), stride, B, ws.idx,
                                          ws.row_seq, ws.unit(), ws.inv_rms, d, eps);
  else
    k_row_rms<uint16_t><<<grid, 256, 0, s>>>(static_cast<const uint16_t*>(x), stride, B, ws.idx,
                                             ws.row_seq, ws.unit(), ws.inv_rms, d, eps);
  return hipGetLastError();
}

// Gather: Hc[r, :] = hidden_g[idx[r], :] and HcT[:, col_off + r] for the unit's
// rows r < N (g = row_seq[r] / B: the row's sample, hidden_g = hidden + g *
// stride); zeros for N <= r < N_pad.  Both are slab-major (Hc with RP rows
// per slab, HcT with d), so each 64x64 tile of either is 8 KB of contiguous
// memory; the tiles are staged in LDS for the transposed copy.  With `gamma`, `hidden` holds the pre-norm activations and
// the gathered row is the final RMSNorm bf16(x * inv_rms[r] * gamma) (fp32
// arithmetic, one rounding to bfloat16).  fp32 inputs are rounded to bf16
// first (load_bf16x8), then treated the same way.
template <typename T>
__global__ __launch_bounds__(256) void k_gather(const T* __restrict__ hidden,
                                                int64_t stride, int B,
                                                const int32_t* __restrict__ idx,
                                                const int32_t* __restrict__ row_seq,
                                                const SampleMeta* __restrict__ meta,
                                                const float* __restrict__ gamma,
                                                const float* __restrict__ inv_rms,
                                                uint16_t* __restrict__ Hc,
                                                uint16_t* __restrict__ HcT, int d, int64_t RP) {
  __shared__ uint16_t tile[64][72];
  const int r0 = blockIdx.x * 64;
  if (r0 >= meta->n_rows_pad) return;
  const int N = meta->n_rows;
  const int coff = meta->col_off;
  const int c0 = blockIdx.y * 64;
  const int tid = threadIdx.x;
#pragma unroll
  for (int it = 0; it < 2; ++it) {
    const int q = tid + it * 256;
    const int row = q >> 3, ch = q & 7;
    const int r = r0 + row;
    uint4 v = make_uint4(0, 0, 0, 0);
    if (r < N) {
      const T* src = hidden + (int64_t)(row_seq[r] / B) * stride + (int64_t)idx[r] * d;
      v = load_bf16x8(src + c0 + ch * 8);
      if (gamma) {
        const float ir = inv_rms[r];
        const float4 g0 = *reinterpret_cast<const float4*>(gamma + c0 + ch * 8);
        const float4 g1 = *reinterpret_cast<const float4*>(gamma + c0 + ch * 8 + 4);
        const float gg[8] = {g0.x, g0.y, g0.z, g0.w, g1.x, g1.y, g1.z, g1.w};
        uint32_t a[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const float lo = __uint_as_float(a[e] << 16), hi = __uint_as_float(a[e] & 0xFFFF0000u);
          a[e] = pack_bf16x2(lo * ir * gg[2 * e], hi * ir * gg[2 * e + 1]);
        }
        v = make_uint4(a[0], a[1], a[2], a[3]);
      }
    }
    *reinterpret_cast<uint4*>(Hc + slab_index(RP, r, c0 + ch * 8)) = v;
    *reinterpret_cast<uint4*>(&tile[row][ch * 8]) = v;
  }
  __syncthreads();
#pragma unroll
  for (int it = 0; it < 2; ++it) {
    const int q = tid + it * 256;
    const int c = q >> 3, rch = q & 7;
    uint32_t w[4];
#pragma unroll
    for (int e = 0; e < 4; ++e)
      w[e] = (uint32_t)tile[rch * 8 + 2 * e][c] | ((uint32_t)tile[rch * 8 + 2 * e + 1][c] << 16);
    *reinterpret_cast<uint4*>(HcT + slab_index(d, c0 + c, (int64_t)coff + r0 + rch * 8)) =
        make_uint4(w[0], w[1], w[2], w[3]);
  }
}

hipError_t launch_gather(const void* hidden, bool f32, int64_t stride, int B, const float* gamma,
                         const Workspace& ws, int d, hipStream_t s) {
  dim3 grid((unsigned)(ws.RP / 64), (unsigned)(d / 64));
  if (f32)
    k_gather<float><<<grid, 256, 0, s>>>(static_cast<const float*>(hidden), stride, B, ws.idx,
                                         ws.row_seq, ws.unit(), gamma, ws.inv_rms, ws.Hc, ws.HcT,
                                         d, ws.RP);
  else
    k_gather<uint16_t><<<grid, 256, 0, s>>>(static_cast<const uint16_t*>(hidden), stride, B,
                                            ws.idx, ws.row_seq, ws.unit(), gamma, ws.inv_rms,
                                            ws.Hc, ws.HcT, d, ws.RP);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// W_head [d, V] -> WT [V, d] (row-major) and, unless Wk is NULL, Wk: W in
// slab-major order with d rows per slab (the dX GEMM's operand; each 64x64
// tile is 8 KB of contiguous memory there).  64x64 tiles through LDS; fp32 W
// is rounded to bf16 as it is read.
template <typename T>
__global__ __launch_bounds__(256) void k_transpose_w(const T* __restrict__ W,
                                                     uint16_t* __restrict__ WT,
                                                     uint16_t* __restrict__ Wk, int d, int V) {
  __shared__ uint16_t tile[64][72];
  const int v0 = blockIdx.x * 64, k0 = blockIdx.y * 64;
  const int tid = threadIdx.x;
#pragma unroll
  for (int it = 0; it < 2; ++it) {
    const int q = tid + it * 256;
    const int kr = q >> 3, ch = q & 7;
    const uint4 v = load_bf16x8(W + (int64_t)(k0 + kr) * V + v0 + ch * 8);
    *reinterpret_cast<uint4*>(&tile[kr][ch * 8]) = v;
    if (Wk) *reinterpret_cast<uint4*>(Wk + slab_index(d, k0 + kr, v0 + ch * 8)) = v;
  }
  __syncthreads();
#pragma unroll
  for (int it = 0; it < 2; ++it) {
    const int q = tid + it * 256;
    const int v = q >> 3, kch = q & 7;
    uint32_t w[4];
#pragma unroll
    for (int e = 0; e < 4; ++e)
      w[e] = (uint32_t)tile[kch * 8 + 2 * e][v] | ((uint32_t)tile[kch * 8 + 2 * e + 1][v] << 16);
    *reinterpret_cast<uint4*>(WT + (int64_t)(v0 + v) * d + k0 + kch * 8) =
        make_uint4(w[0], w[1], w[2], w[3]);
  }
}

hipError_t launch_transpose_w(const void* W, bool f32, uint16_t* WT, uint16_t* Wk, int d, int V,
                              hipStream_t s) {
  dim3 grid((unsigned)(V / 64), (unsigned)(d / 64));
  if (f32)
    k_transpose_w<float><<<grid, 256, 0, s>>>(static_cast<const float*>(W), WT, Wk, d, V);
  else
    k_transpose_w<uint16_t><<<grid, 256, 0, s>>>(static_cast<const uint16_t*>(W), WT, Wk, d, V);
  return hipGetLastError();
}

}  // namespace bgpo
