// The bf16 MFMA GEMM core for gfx950 and its epilogues.
//
// Every contraction of the ELBO head is written in one form,
//     C[m][n] = sum_k A[m][k] * B[n][k],
// B always K-contiguous, so that its 16-byte vectors match the MFMA operand
// layout directly:
//   forward               Z^T[v][row] = WT[v][:] . Hc[row][:]     (K = d)
//   dX (split over V)     dX^T[c][row] = W[c][:] . dZ[row][:]     (K = V)
//   dW                    dW^T[v][c]  += dZ[:][v] . HcT[c][:]     (K = rows)
// Operand layouts: the head weights (WT, and W in the dX GEMM) are
// row-major; the per-unit operands (Hc, dZ, HcT) are K-slab-major: element
// (r, k) of a matrix with R rows per slab sits at ((k / 64) R + r) 64 +
// k % 64, so the 64-deep slab of a 256-row panel that one pipeline stage
// loads is 32 KB of contiguous memory.  (Row-major, with rows V or the row
// count long, each slab of a panel touched 256 rows far apart, and the loads
// ran slower.)  The dW GEMM reads dZ, the dX GEMM's operand, as its A with
// the roles of the two indices swapped (M = vocabulary contiguous within a
// slab, K = rows): its fragments come from the transposing LDS read, so the
// exponentials are kept in one layout only.
// The logits are produced as Z^T (vocabulary along M) so that each lane holds
// vocabulary entries of few rows: the per-row max / sum-exp reductions are
// in-lane plus lane swaps.  dX and dW are produced transposed and stored
// transposed, so that a lane's 4 accumulator values land in one 16-byte store.
//
// Scheduling: a persistent grid of one workgroup per compute unit walks the
// tile list in bands of M tiles; consecutive tiles (sharing operand panels)
// go to workgroups of the same XCD (workgroup w runs on XCD w mod 8), so the
// shared panels are served from that XCD's L2.
//
// Pipeline: a two-stage LDS ring of 64-deep K slabs, filled by direct
// buffer-to-LDS loads (no staging registers); a stage is refilled with the
// slab two ahead as soon as the barrier that ends its last use has passed.
// LDS rows are XOR-swizzled in 16-byte chunks so that fragment reads of
// consecutive rows hit distinct banks.
//
// k_gemm4w: four waves of 128x128 on 16x16x32 MFMAs in inline assembly with
// accumulators in AGPRs, hand-ordered (see below).
#include "common.hpp"
#include "internal.hpp"

#include <string.h>

namespace bgpo {

enum EpiKind { EPI_FWD = 0, EPI_FWDU = 1, EPI_F32_STORE = 2, EPI_F32_ACCUM = 3, EPI_DZ = 4 };

// Layouts of the A operand.  A_ROW: row-major, lda elements per row (W^T in
// the forward).  A_KSLAB: slab-major over K, element (m, k) at
// ((k / 64) lda + m) 64 + k % 64 with lda = M rows per slab (W in the dX
// GEMM: a tile's K slab is one contiguous run of 128-byte rows instead of
// rows a whole vocabulary apart).  A_MSLAB: the transpose stored slab-major,
// element (m, k) at ((m / 64) lda + k) 64 + m % 64 with lda = K rows per slab
// (dZ as the dW GEMM's A): M is contiguous, so its fragments are read with
// the transposing LDS read.
enum ALayout { A_ROW = 0, A_MSLAB = 1, A_KSLAB = 2 };

struct GemmParams {
  const uint16_t* A;
  int64_t lda;               // A_ROW: elements per row; A_KSLAB: rows (M) per slab;
                             // A_MSLAB: rows (K) per slab
  const uint16_t* B;
  int64_t ldb;               // rows per slab (B is always slab-major)
  int dyn_boff;              // B starts at row meta->col_off (the unit's rows of dZ)
  int M, N, K;               // static extents
  int dyn_m, dyn_n, dyn_k;   // extents taken from the device sample metadata
  int dyn_split;             // K split taken from the metadata (dX)
  int n_split;               // K split count
  int64_t k_split;           // K per split (multiple of BK)
  int group_m;              // tile order: bands of group_m M tiles, walking along N
                             // (1 = N tiles consecutive, tilesM = M tiles consecutive)
  const SampleMeta* meta;
  // epilogue operands
  float* out;                // F32 store / accumulate target
  int64_t ldo, split_stride;
  float* part_m;             // FWD: per-128-vocabulary-slice (max, sum) partials [M/WM][ldp]
  float* part_s;
  int64_t ldp;
  uint16_t* dZ;              // FWDU: exponentials u, rows from the unit's col_off; DZ: the
  int64_t ldz;               // chunk's dZ (slab-major, ldz rows per slab)
  const float* lse2;         // DZ: per-row log2-sum-exp2, gradient scale and target id
  const float* rscale;
  const int32_t* rtgt;
  const float* ztgt;         // FWDU: per-row target logit (the exponent reference)
  int v0;                    // DZ: vocabulary id of row 0 of A (the chunk's first id)
};

template <int BM, int BN, int BK, int WM, int WN>
struct Cfg {
  static constexpr int NWM = BM / WM, NWN = BN / WN;
  static constexpr int NWAVES = NWM * NWN;
  static constexpr int NT = NWAVES * 64;
  static constexpr int KCH = BK / 8;                  // 16-byte chunks per LDS row
  static_assert(BM * KCH % NT == 0 && BN * KCH % NT == 0, "load split");
  static_assert(KCH == 8, "64-deep slabs: one 128-byte line per LDS row");
  // 16-byte chunk c of LDS row r is stored at chunk c ^ swz(r): 16 consecutive
  // rows spread over 256 bytes (pairs of rows share a key, and consecutive
  // rows already alternate 128-byte halves)
  __device__ static __forceinline__ int swz(int row) { return (row >> 1) % KCH; }
};

// The chunk swizzle of an A_MSLAB operand in LDS: 16-byte chunk c (8 M ids)
// of K row k sits at chunk c ^ mslab_swz(k).  A transposing fragment read
// takes 32 bytes (two chunks) of each of 16 K rows: rows 8 g + e (e < 4) of
// lane groups g = 0, 1, and those rows + 4.  The XOR term moves the four rows
// of one group (bits 0 and 1 of k) to distinct 32-byte segments, and, among
// rows of one parity (one 128-byte half of the 256 bytes that the banks
// span), the rows of the two groups (bit 3) too; it is even, so a pair of
// chunks stays adjacent, and it ignores bit 2, so the rows k and k + 4 of
// the two reads share it.
__device__ __forceinline__ int mslab_swz(int k) {
  return 2 * (((k ^ (k >> 3)) & 1) | (k & 2));
}

// One buffer load of 16 bytes per lane straight into LDS (lds_dst + 16 per
// lane), as inline assembly.  The compiler's own form of this load makes it
// wait for all outstanding loads before every LDS read that it cannot prove
// independent of them (the transposing reads of an A_MSLAB operand, which
// carry no type information); the ring's explicit waits already order them.
// The LDS-DMA load reads M0 one wait state after the scalar write at the
// earliest (the s_nop; the compiler does not see inside the statement).
__device__ __forceinline__ void lds_load16_asm(__amdgpu_buffer_rsrc_t rsrc, uint32_t voff,
                                               uint32_t soff, const void* lds_dst) {
  const uint32_t la = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) const void*)lds_dst;
  asm volatile("s_mov_b32 m0, %3\n\ts_nop 0\n\tbuffer_load_dwordx4 %0, %1, %2 offen lds"
               :
               : "v"(voff), "s"(rsrc), "s"(soff), "s"(__builtin_amdgcn_readfirstlane(la))
               : "memory", "m0");
}

// s_waitcnt vmcnt(N) with the other counters left alone (gfx9 encoding: vmcnt
// in bits 3:0 and 15:14, expcnt 6:4, lgkmcnt 11:8).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// A per-row value for each of a lane's 8 accumulator rows, row
// nw + 16 j + (lane % 16) for j = 0 .. 7: the wave's 128 rows in two
// coalesced loads (lane l takes rows nw + l and nw + 64 + l, f of the loaded
// value, or `fill` at rows not below n_valid), then lane shuffles.  With one
// load per row the compiler issued and waited for the eight loads one after
// the other, and where a row's value was first used inside a conditional
// block it waited again there for every outstanding store.  (Clamped
// unconditional loads, to have both in flight under one wait, changed the
// register allocation: spill reloads then waited inside the column loop.)
template <typename T, typename F>
__device__ __forceinline__ void rows_of_lane(const T* src, int nw, int n_valid, int lane, T fill,
                                             F f, T (&out)[8]) {
  const int na = nw + lane, nb = nw + 64 + lane;
  const T a = na < n_valid ? f(src[na]) : fill;
  const T b = nb < n_valid ? f(src[nb]) : fill;
#pragma unroll
  for (int j = 0; j < 8; ++j) out[j] = __shfl(j < 4 ? a : b, 16 * (j & 3) + (lane & 15), 64);
}

// One 16-byte bf16 store per lane for two vertically adjacent 16x16 blocks
// (blocks i and i + 1 of one column block): lane l holds 4 consecutive ids
// 4 (l / 16) .. + 3 of each (lo: block i, hi: block i + 1, packed bf16).
// v_permlane16_swap trades the hi values of the even 16-lane rows for the lo
// values of the odd rows, so that a lane of an even row holds ids 8 r .. 8 r
// + 7 of block i and a lane of an odd row those of block i + 1 (r = l / 32):
// 8 consecutive ids of one accumulator row, at tile id 16 (i + (l / 16) % 2) +
// 8 (l / 32).  (Measured against one 8-byte store per block: forward GEMM
// 2-4 % faster.)
__device__ __forceinline__ uint4 pair_rows16(uint2 lo, uint2 hi) {
  const auto sx = __builtin_amdgcn_permlane16_swap(lo.x, hi.x, false, false);
  const auto sy = __builtin_amdgcn_permlane16_swap(lo.y, hi.y, false, false);
  return make_uint4(sx[0], sy[0], sx[1], sy[1]);
}

// ---------------------------------------------------------------------------
// The production kernel: one wave per SIMD on v_mfma_f32_16x16x32_bf16.
//
// Lane l of a 16x16x32 MFMA holds A[m = l % 16][k = 8 (l / 16) + t] and
// B[k = 8 (l / 16) + t][n = l % 16] (t = 0..7: one 16-byte LDS chunk each)
// and accumulates C[m = 4 (l / 16) + e][n = l % 16] (e = 0..3).  A 256x256
// block tile is split over four waves of 128x128, so each wave holds 8x8
// accumulator blocks (all 256 AGPRs) and reads, per 64-deep slab, its 128 rows
// of A and of B once: a third less LDS traffic per MFMA than eight waves of
// 128x64, and the 16x16x32 form moves half the accumulator bytes per FLOP of
// the 32x32x16 form, which keeps the clock higher under the power cap.
//
// The MFMAs are inline assembly on accumulators tied to AGPRs ("+a"): with
// the compiler's own MFMA builtins on 256 accumulator registers the register
// allocator moved accumulators through spare AGPRs on every iteration.  The
// instruction order is fixed by hand: per 32-deep sub-step 64 MFMAs, with one
// fragment read of the next sub-step after every fourth MFMA (both operands'
// fragments double-buffered in VGPRs) and, in the sub-step after a slab
// barrier, one slab load after every fourth as well.  Because the compiler
// does not see these MFMAs as such, the code pads the two hazards it would
// otherwise cover: accumulator writes before the first MFMA reads them, and
// the last MFMAs' results before the epilogue reads them.
typedef float f32x4 __attribute__((ext_vector_type(4)));

#define BGPO_MFMA16(acc, a, b) \
  asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, %0" : "+a"(acc) : "v"(a), "v"(b))

// fp32 store of a wave tile of 16x16 accumulator blocks, transposed: element
// (m, n) goes to out[n * ldo + m], so a lane's 4 values of one block
// (m = 4 (lane / 16) .. + 3 of one n) are one 16-byte store.  ACCUM: add to
// the current values (read first, one column block at a time).  M is a
// multiple of 4 (the vocabulary and hidden sizes are multiples of 64).
template <bool ACCUM, bool FULL, int TM, int TN>
__device__ __forceinline__ void epi_f32_16t(const f32x4 (&acc)[TM][TN], float* outb, int64_t ldo,
                                            int mw, int nw, int lane, int M, int N) {
  const int mlane = 4 * (lane >> 4);
#pragma unroll
  for (int j = 0; j < TN; ++j) {
    const int n = nw + 16 * j + (lane & 15);
    float* col = outb + (int64_t)n * ldo + mw + mlane;
    f32x4 old[TM];
    if constexpr (ACCUM) {
#pragma unroll
      for (int i = 0; i < TM; ++i)
        old[i] = (FULL || (mw + 16 * i + mlane < M && n < N))
                     ? *reinterpret_cast<const f32x4*>(col + 16 * i)
                     : (f32x4){0.f, 0.f, 0.f, 0.f};
    }
#pragma unroll
    for (int i = 0; i < TM; ++i)
      if (FULL || (mw + 16 * i + mlane < M && n < N))
        *reinterpret_cast<f32x4*>(col + 16 * i) = ACCUM ? old[i] + acc[i][j] : acc[i][j];
    __builtin_amdgcn_sched_barrier(0);
  }
}

template <int EPI, int AL, int BM, int BN, int BK, int STAGES>
__global__ __launch_bounds__(256, 1) void k_gemm4w(GemmParams p) {
#if defined(__HIP_DEVICE_COMPILE__)  // the host pass needs only the signature
  constexpr int WM = 128, WN = 128;
  using C = Cfg<BM, BN, BK, WM, WN>;
  constexpr int NT = C::NT, KCH = C::KCH;
  constexpr int TM = WM / 16, TN = WN / 16;
  // 64-deep slabs hold two 32-deep MFMA sub-steps between barriers
  static_assert(C::NWAVES == 4 && BK == 64, "four waves, 64-deep slabs");
  // A is row-major (W^T, W) or M-slab-major (dZ, with transposing fragment
  // reads); B is always K-slab-major
  constexpr bool kMSlabA = AL == A_MSLAB, kKSlabA = AL == A_KSLAB;
  static_assert(!kMSlabA || BM / 64 == C::NWAVES, "one 64-row M slab of A per wave");
  __shared__ uint4 smem[STAGES * (BM + BN) * KCH];
  uint4* As = smem;                           // [STAGES][BM][KCH]
  uint4* Bs = smem + STAGES * BM * KCH;       // [STAGES][BN][KCH]

  const int tid = threadIdx.x;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave-uniform, kept in an SGPR
  const int wm = wave / C::NWN, wn = wave % C::NWN;

  int M = p.M, N = p.N, K = p.K, n_valid = p.N;
  if (p.dyn_m) { M = p.meta->n_rows_pad; n_valid = p.meta->n_rows; }
  if (p.dyn_n) { N = p.meta->n_rows_pad; n_valid = p.meta->n_rows; }
  if (p.dyn_k) K = p.meta->col_end;    // batched dW: all samples' columns (multiple of 64)
  // first row of the unit in dZ (EPI_FWDU), read once into a scalar register
  const int zt_col = EPI == EPI_FWDU ? __builtin_amdgcn_readfirstlane(p.meta->col_off) : 0;
  // first row of B (the unit's rows of a dZ shared by a dW batch)
  const int b_row0 = p.dyn_boff ? __builtin_amdgcn_readfirstlane(p.meta->col_off) : 0;
  int n_split = p.n_split;
  int64_t k_split = p.k_split;
  if (p.dyn_split) {
    n_split = p.meta->dx_split;
    k_split = (int64_t)p.meta->dx_kslab * 64;   // whole 64-deep slabs
  }
  if (EPI == EPI_F32_ACCUM && K == 0) return;   // nothing to add
  // The tile walk in 32-bit wave-uniform (scalar) arithmetic: tile counts
  // stay below 2^30 for every launch (tiles of M and N below 2^12 and 2^14,
  // at most 16 splits; the test hook checks its own).
  const uint32_t tilesM = __builtin_amdgcn_readfirstlane((M + BM - 1) / BM);
  const uint32_t tilesN = __builtin_amdgcn_readfirstlane((N + BN - 1) / BN);
  const uint32_t per_split = tilesM * tilesN;
  const uint32_t total = __builtin_amdgcn_readfirstlane(per_split * (uint32_t)n_split);
  const uint32_t GM = __builtin_amdgcn_readfirstlane(max(1, min(p.group_m, (int)tilesM)));
  const uint32_t band_tiles = GM * tilesN;
  const uint32_t G = gridDim.x;
  const uint32_t w = blockIdx.x;
  const uint32_t xcd_slot = G % 8 == 0 ? (w % 8) * (G / 8) + w / 8 : w;

  for (uint32_t t = xcd_slot; t < total; t += G) {
    // the lane index, recomputed every tile from the execution mask (volatile
    // asm, so neither it nor the addresses formed from it are hoisted out of
    // the tile loop: with all 256 AGPRs holding accumulators, hoisted values
    // are spilled, and their reload at the loop head waits for every
    // outstanding store of the previous tile)
    int lane_t;
    asm volatile("v_mbcnt_lo_u32_b32 %0, -1, 0\n\tv_mbcnt_hi_u32_b32 %0, -1, %0" : "=v"(lane_t));
    const int lane = lane_t;
    int mt, nt, split;
    {
      // bands of GM M tiles walk along N: 32 consecutive tiles (one XCD's
      // share of a round) cover GM M tiles x 32 / GM N tiles
      const uint32_t sp = __builtin_amdgcn_readfirstlane(t / per_split);
      const uint32_t r = t - sp * per_split;
      const uint32_t band = __builtin_amdgcn_readfirstlane(r / band_tiles);
      const uint32_t gm = min(GM, tilesM - band * GM);
      const uint32_t idx = r - band * band_tiles;
      const uint32_t q = __builtin_amdgcn_readfirstlane(idx / gm);
      split = (int)sp;
      mt = (int)(band * GM + (idx - q * gm));
      nt = (int)q;
    }
    const int m0 = mt * BM, n0 = nt * BN;
    const int64_t kb = (int64_t)split * k_split;
    const int64_t ke = min((int64_t)K, kb + k_split);
    const int nk = ke > kb ? (int)((ke - kb) / BK) : 0;

    // accumulator element (i, j, e) sits at
    //   m = mw + 16 i + 4 (lane >> 4) + e,  n = nw + 16 j + (lane & 15)
    const int mw = m0 + wm * WM, nw = n0 + wn * WN;
    const int mlane = 4 * (lane >> 4);
    f32x4 acc[TM][TN];
    // dW accumulates in place: a full tile starts from the current output
    // (loaded straight into the accumulator registers before the slab loads,
    // so the wait for the first slab covers them) and ends with plain stores;
    // a partial tile starts from zero and adds in its epilogue
    const bool preload = EPI == EPI_F32_ACCUM && m0 + BM <= M && n0 + BN <= N;
    if (preload) {
      const float* src = p.out + (int64_t)split * p.split_stride + (int64_t)(nw + (lane & 15)) * p.ldo +
                         mw + mlane;
#pragma unroll
      for (int j = 0; j < TN; ++j)
#pragma unroll
        for (int i = 0; i < TM; ++i)
          asm volatile("global_load_dwordx4 %0, %1, off"
                       : "=a"(acc[i][j])
                       : "v"(src + (int64_t)16 * j * p.ldo + 16 * i));
    } else {
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[i][j] = (f32x4){0.f, 0.f, 0.f, 0.f};
    }
    asm volatile("s_nop 4");   // accumulator writes land before the first MFMA reads them

    // Operand panels as buffer resources; each load instruction moves 64
    // lanes x 16 bytes straight into LDS, the XOR swizzle applied on the
    // global side; rows past the matrix are clamped to its last row.  A
    // row-major panel is one descriptor with the slab's K offset as the
    // scalar offset; a slab-major panel gets a descriptor per slab (its
    // slabs lie rows-per-slab x 128 bytes apart, beyond 32-bit offsets), with
    // rows 128 bytes apart inside it.
    const char* const a_tile = reinterpret_cast<const char*>(
        p.A + (kMSlabA   ? (int64_t)(m0 / 64) * p.lda * 64
               : kKSlabA ? (int64_t)m0 * 64
                         : (int64_t)m0 * p.lda));
    const char* const b_tile = reinterpret_cast<const char*>(p.B + ((int64_t)n0 + b_row0) * 64);
    const int64_t a_slab = p.lda * 128, b_slab = p.ldb * 128;   // bytes per slab (slab-major)
    const int a_row = (int)p.lda * 2;                           // bytes per row (A_ROW)
    const __amdgpu_buffer_rsrc_t a_rsrc =
        __builtin_amdgcn_make_buffer_rsrc((void*)a_tile, (short)0, 0x7FFFFFFF, 0x00020000);
    constexpr int RPI = 64 / KCH;                        // rows per load instruction
    constexpr int A_INS = BM / RPI / C::NWAVES, B_INS = BN / RPI / C::NWAVES;
    static_assert(A_INS + B_INS == BK / 4, "one slab load per 256 / BK MFMAs");
    uint32_t a_voff[A_INS], b_voff[B_INS];
    // A_MSLAB: wave w loads M slab w of the tile (the matrix's last slab for
    // slabs past M), K rows 8 q .. 8 q + 7 of it per instruction q, into
    // LDS [M slab][K row][8 chunks of 8 M ids], chunk-swizzled by K row
    const int64_t a_wslab =
        kMSlabA ? (int64_t)(min(m0 / 64 + wave, (M + 63) / 64 - 1) - m0 / 64) * a_slab : 0;
#pragma unroll
    for (int q = 0; q < A_INS; ++q) {
      if constexpr (kMSlabA) {
        const int k = 8 * q + lane / KCH;
        a_voff[q] = (uint32_t)(k * 128 + ((lane % KCH) ^ mslab_swz(k)) * 16);
      } else {
        const int g = wave * A_INS + q, row = g * RPI + lane / KCH;
        const int c = (lane % KCH) ^ C::swz(row);
        const int rr = min(m0 + row, M - 1) - m0;
        a_voff[q] = (uint32_t)(rr * (kKSlabA ? 128 : a_row) + c * 16);
      }
    }
#pragma unroll
    for (int q = 0; q < B_INS; ++q) {
      const int g = wave * B_INS + q, row = g * RPI + lane / KCH;
      const int c = (lane % KCH) ^ C::swz(row);
      const int rr = min(n0 + row, N - 1) - n0;
      b_voff[q] = (uint32_t)(rr * 128 + c * 16);
    }
    if (nk > 0) {
      // S-stage ring of K slabs: slab q lives in stage q % S,
      // slab c + S is loaded into slab c's stage right after the barrier that
      // ends slab c, and slabs past the tile's K range re-load its last slab.
      constexpr int NINS = A_INS + B_INS;
      auto lds_load = [&](__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff, uint4* dst) {
        if constexpr (kMSlabA)
          lds_load16_asm(r, voff, soff, dst);
        else
          __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (__attribute__((address_space(3))) void*)dst, 16,
                                                   voff, soff, 0, 0);
      };
      auto issue_one = [&](int q, int stage, int e) {   // load instruction e of slab q
        const int qc = min(q, nk - 1);
        const int64_t ks = kb / BK + qc;                  // slab index in K
        if (e < A_INS) {
          uint4* dst = As + stage * BM * KCH + (wave * A_INS + e) * 64;
          if constexpr (kMSlabA) {
            // K slab ks of the wave's M slab: 64 rows of 128 bytes
            lds_load(__builtin_amdgcn_make_buffer_rsrc((void*)(a_tile + a_wslab + ks * 8192), (short)0,
                                                       0x7FFFFFFF, 0x00020000),
                     a_voff[e], 0, dst);
          } else if constexpr (kKSlabA) {
            lds_load(__builtin_amdgcn_make_buffer_rsrc((void*)(a_tile + ks * a_slab), (short)0,
                                                       0x7FFFFFFF, 0x00020000),
                     a_voff[e], 0, dst);
          } else {
            lds_load(a_rsrc, a_voff[e], (uint32_t)(ks * BK * 2), dst);
          }
        } else {
          uint4* dst = Bs + stage * BN * KCH + (wave * B_INS + e - A_INS) * 64;
          lds_load(__builtin_amdgcn_make_buffer_rsrc((void*)(b_tile + ks * b_slab), (short)0, 0x7FFFFFFF,
                                                     0x00020000),
                   b_voff[e - A_INS], 0, dst);
        }
      };
#pragma unroll
      for (int q = 0; q < STAGES; ++q)
#pragma unroll
        for (int e = 0; e < NINS; ++e) issue_one(q, q, e);
      wait_vmcnt<NINS * (STAGES - 1)>();
      __builtin_amdgcn_s_barrier();

      bf16x8 fa[2][TM], fb[2][TN];
      const int arow = wm * WM + (lane & 15), brow = wn * WN + (lane & 15);
      // fragment r of 32-deep sub-step ks of stage st: B block r for r < TN,
      // else A block r - TN
      auto rd = [&](bf16x8 (&da)[TM], bf16x8 (&db)[TN], int st, int ks, int r) {
        const int ch = ks * 4 + (lane >> 4);
        if (r < TN) {
          const int row = brow + 16 * r;
          db[r] = __builtin_bit_cast(bf16x8, Bs[st * BN * KCH + row * KCH + (ch ^ C::swz(row))]);
        } else if constexpr (kMSlabA) {
          // A[m][k .. k + 7] of M id m = 16 i + lane % 16 of the wave's rows,
          // k = 32 ks + 8 (lane / 16), from LDS [M slab][K row][M]: two
          // transposing reads, each returning to lane 4 q + t of a 16-lane
          // group element t of the 8 bytes that lanes q, q + 4, q + 8, q + 12
          // address; lane 4 e + q of group g addresses K row 8 g + e (+ 4)
          // at M ids 16 i + 4 q .. + 3
          const int i = r - TN, g = lane >> 4, jl = lane & 15;
          const int kr = 32 * ks + 8 * g + (jl >> 2);
          const int mm = wm * WM + 16 * i + 4 * (jl & 3);   // M id within the tile
          const char* base = reinterpret_cast<const char*>(As + st * BM * KCH) + (mm >> 6) * 8192 +
                             (((mm & 63) >> 3) ^ mslab_swz(kr)) * 16 + (mm & 7) * 2;
          typedef short v4s __attribute__((ext_vector_type(4)));
          typedef __attribute__((address_space(3))) v4s lds_v4s;
          const v4s lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s*)(base + kr * 128));
          const v4s hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s*)(base + (kr + 4) * 128));
          const uint2 l2 = __builtin_bit_cast(uint2, lo), h2 = __builtin_bit_cast(uint2, hi);
          da[i] = __builtin_bit_cast(bf16x8, make_uint4(l2.x, l2.y, h2.x, h2.y));
        } else {
          const int row = arow + 16 * (r - TN);
          da[r - TN] =
              __builtin_bit_cast(bf16x8, As[st * BM * KCH + row * KCH + (ch ^ C::swz(row))]);
        }
      };
      // one sub-step on fragment set h: its 64 MFMAs, the reads of sub-step
      // (nst, nks) into set 1 - h and, with `loads`, slab lq into stage lst.
      // The sub-step before a barrier issues its 16 reads after every third
      // of its first 48 MFMAs, so that the reads are complete when the wave
      // reaches the barrier's wait (measured 1 % faster than reads spread to
      // the last MFMA); the other sub-step reads after every fourth.
      constexpr int LEVERY = TM * TN / NINS;   // MFMAs per slab load
      auto step = [&](int h, int nst, int nks, bool loads, int lq, int lst, bool pre) {
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int j = 0; j < TN; ++j) {
            const int m = i * TN + j;
            BGPO_MFMA16(acc[i][j], fa[h][i], fb[h][j]);
            if (loads && m % LEVERY == 1) issue_one(lq, lst, m / LEVERY);
            if (pre) {
              if (m % 3 == 0 && m / 3 < TM + TN) rd(fa[1 - h], fb[1 - h], nst, nks, m / 3);
            } else if ((m & 3) == 3) {
              rd(fa[1 - h], fb[1 - h], nst, nks, m >> 2);
            }
            __builtin_amdgcn_sched_barrier(0);
          }
      };
#pragma unroll
      for (int r = 0; r < TM + TN; ++r) rd(fa[0], fb[0], 0, 0, r);
      // every slab, the last one included, runs the same code (the last
      // one's reads and loads fetch data nobody uses), so the accumulators
      // stay in their registers across the whole loop
      for (int kt = 0; kt < nk; ++kt) {
        const int cur = kt % STAGES;
        step(0, cur, 1, false, 0, 0, true);
        // slab kt + 1 landed (own loads) and, after the barrier, every wave
        // is done with stage `cur`: refill it with slab kt + S during the
        // second sub-step, which also reads slab kt + 1's first fragments
        wait_vmcnt<NINS * (STAGES - 2)>();
        __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0)
        __builtin_amdgcn_s_barrier();
        __builtin_amdgcn_sched_barrier(0);
        step(1, (kt + 1) % STAGES, 0, true, kt + STAGES, cur, false);
      }
      // drain the ring (outstanding re-loads) before the epilogue may reuse LDS
      __builtin_amdgcn_s_waitcnt(0);
      __builtin_amdgcn_s_barrier();
    }
    asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7");   // the last MFMAs' results land

    // ---------------- epilogues ----------------
    if constexpr (EPI == EPI_FWD || EPI == EPI_FWDU) {
      // Per (row, 128-entry vocabulary slice of this wave): max m and sum of
      // 2^(z log2e - m), in log2 units, written to the partials (the slice of
      // wave row wm is partial index mw / 128).  A row's 128 entries sit in
      // its lane and the lanes l ^ 16, l ^ 32, l ^ 48.  EPI_FWDU also keeps
      // the exponentials against the row's reference R2 (exp_reference of
      // its target logit), u = 2^(z log2e - m) 2^(m - R2), in bf16, in dZ
      // (rows from the unit's col_off, the layout both backward GEMMs read):
      // dZ is s 2^(R2 - lse2) (u - onehot 2^(lse2 - R2)), so one factor per
      // row makes them the gradient (applied after the GEMMs), and only the
      // target entries change.  A lane's 4 values of a block are 4
      // consecutive vocabulary ids of one row; two blocks' values, traded
      // between lane rows (pair_rows16), are one 16-byte store straight from
      // the registers.  Both variants sum in the same order, so l is
      // bit-identical between them.
      static_assert(WM == kVocabTile, "one partial per wave slice");
      constexpr bool kStore = EPI == EPI_FWDU;
      if (mw + WM > M) {
        // the wave slice crosses the end of the vocabulary: entries past it
        // become -inf, i.e. exponentials 0 (wave-uniform branch)
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int e = 0; e < 4; ++e)
              if (mw + 16 * i + mlane + e >= M) acc[i][j][e] = -INFINITY;
      }
      // one 16-row column block of the wave tile at a time, so that only its
      // 32 values per lane are live outside the accumulators
      const int vt = mw / WM;
      // the wave's partial rows (vt is wave-uniform: a scalar base, 32-bit
      // per-lane offsets)
      float* const pm = p.part_m + (int64_t)vt * p.ldp;
      float* const ps = p.part_s + (int64_t)vt * p.ldp;
      // the references of the lane's 8 rows, loaded before the column blocks
      // so that one wait covers them (padding rows: R2 = 0)
      static_assert(TN == 8, "8 rows per lane");
      float r2v[TN];
      if constexpr (kStore)
        rows_of_lane(p.ztgt, nw, n_valid, lane, 0.f, [](float z) { return exp_reference(z); }, r2v);
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        float mx = -INFINITY;
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int e = 0; e < 4; ++e) mx = fmaxf(mx, acc[i][j][e]);
        mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
        mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
        const float mref = mx > -INFINITY ? mx * kLog2e : 0.f;   // a slice past V has no entries
        float ssum = 0.f;
        const int nl = nw - n0 + 16 * j + (lane & 15);
        // 2^(m - R2): the slice's exponentials against the row's reference
        float fac = 0.f;
        if constexpr (kStore) fac = __builtin_amdgcn_exp2f(mref - r2v[j]);
        static_assert(TM % 2 == 0, "blocks stored in pairs");
#pragma unroll
        for (int i = 0; i < TM; i += 2) {
          uint2 pk[2];
#pragma unroll
          for (int h = 0; h < 2; ++h) {
            float u[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              u[e] = __builtin_amdgcn_exp2f(fmaf(acc[i + h][j][e], kLog2e, -mref));
              ssum += u[e];
            }
            pk[h] = make_uint2(pack_bf16x2(u[0] * fac, u[1] * fac), pack_bf16x2(u[2] * fac, u[3] * fac));
          }
          if constexpr (kStore) {
            // vocabulary ids m .. m + 7 of row n0 + nl (within m's slab)
            const uint4 v = pair_rows16(pk[0], pk[1]);
            const int m = mw + 16 * (i + ((lane >> 4) & 1)) + 8 * (lane >> 5);
            if (n0 + nl < N && m < M)
              *reinterpret_cast<uint4*>(p.dZ + ((int64_t)(m >> 6) * p.ldz + zt_col + n0 + nl) * 64 +
                                        (m & 63)) = v;
          }
        }
        float st = ssum + __shfl_xor(ssum, 16, 64);
        st += __shfl_xor(st, 32, 64);
        const int n = n0 + nl;
        if (lane < 16 && mw < M && n < n_valid) {
          pm[(uint32_t)n] = mref;
          ps[(uint32_t)n] = st;
        }
        __builtin_amdgcn_sched_barrier(0);
      }
    } else if constexpr (EPI == EPI_DZ) {
      // Recompute backward: the tile holds logits z of vocabulary ids
      // v0 + m (M) for rows n (N); each becomes
      //   dZ = s_n (2^(z log2e - lse2_n) - [v0 + m == y_n])
      // in bf16 (RNE), s_n and lse2_n of the row (the derivative of the
      // scaled loss term w.r.t. the logit, Eq. per_step_loss with the
      // gradient scale of the response's bound term); padding rows get exact
      // zeros.  Stored like the forward's exponentials: 16 bytes per lane and
      // pair of blocks straight into the chunk's slab-major dZ, which the dX GEMM reads
      // as its B operand and the dW GEMM as its M-slab-major A operand.
      // the lane's 8 rows' log2-sum-exp2, scale and target (as a tile row
      // index, may be outside), loaded before the column blocks so that one
      // wait covers them
      float l2v[TN], srv[TN];
      int ymv[TN];
      const int ysh = p.v0 + m0;
      rows_of_lane(p.lse2, nw, n_valid, lane, 0.f, [](float v) { return v; }, l2v);
      rows_of_lane(p.rscale, nw, n_valid, lane, 0.f, [](float v) { return v; }, srv);
      rows_of_lane(p.rtgt, nw, n_valid, lane, -1, [ysh](int y) { return y - ysh; }, ymv);
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int nl = nw - n0 + 16 * j + (lane & 15);
        const bool live = n0 + nl < n_valid;
        const float l2 = l2v[j], sr = srv[j];
        const int ym = ymv[j];
#pragma unroll
        for (int i = 0; i < TM; i += 2) {
          uint2 pk[2];
#pragma unroll
          for (int h = 0; h < 2; ++h) {
            const int ml = mw - m0 + 16 * (i + h) + mlane;
            float x[4];
#pragma unroll
            for (int e = 0; e < 4; ++e) {
              const float pz = __builtin_amdgcn_exp2f(fmaf(acc[i + h][j][e], kLog2e, -l2));
              x[e] = live ? sr * (ml + e == ym ? pz - 1.f : pz) : 0.f;
            }
            pk[h] = make_uint2(pack_bf16x2(x[0], x[1]), pack_bf16x2(x[2], x[3]));
          }
          const uint4 v = pair_rows16(pk[0], pk[1]);
          const int m = mw + 16 * (i + ((lane >> 4) & 1)) + 8 * (lane >> 5);
          if (n0 + nl < N && m < M)
            *reinterpret_cast<uint4*>(p.dZ + ((int64_t)(m >> 6) * p.ldz + n0 + nl) * 64 + (m & 63)) = v;
        }
        __builtin_amdgcn_sched_barrier(0);
      }
    } else {
      // fp32 store of the tile, transposed (dX partials, or a full dW tile
      // that started from its previous value), or read-modify-write of a
      // partial dW tile
      float* outb = p.out + (int64_t)split * p.split_stride;
      if (m0 + BM <= M && n0 + BN <= N) epi_f32_16t<false, true, TM, TN>(acc, outb, p.ldo, mw, nw, lane, M, N);
      else epi_f32_16t<EPI == EPI_F32_ACCUM, false, TM, TN>(acc, outb, p.ldo, mw, nw, lane, M, N);
    }
    __syncthreads();
  }
#endif
}

// Tile configuration of the production kernels (k_gemm4w): 256x256 block
// tile, K slab 64 in a 2-stage LDS ring, four waves of 128x128, 256-byte LDS
// swizzle.
#define BGPO_TILE4 256, 256, 64, 2
constexpr int kGemmThreads4 = 256;
// band heights of the tile walk (bands of M tiles walking along N),
// measured at the LLaDA head shape: dW and dX fastest with bands of 8, the
// forward GEMM with bands of 4 (2 or 8: 2 % slower, 16: 7 %)
constexpr int kGroupMdW = 8;
constexpr int kGroupMdX = 8;
constexpr int kGroupMFwd = 4;

static GemmParams base_params() {
  GemmParams p;
  memset(&p, 0, sizeof(p));
  p.n_split = 1;
  p.k_split = INT64_MAX / 4;
  p.group_m = 1;
  return p;
}

hipError_t launch_gemm_fwd(const Workspace& ws, int d, int V, int grid, bool store_u,
                           hipStream_t s) {
  GemmParams p = base_params();
  p.A = ws.WT; p.lda = d;
  p.B = ws.Hc; p.ldb = ws.RP;
  p.M = V; p.K = d; p.dyn_n = 1; p.meta = ws.unit();
  p.k_split = d;
  p.part_m = ws.part_m; p.part_s = ws.part_s; p.ldp = ws.RP;
  p.group_m = kGroupMFwd;
  if (store_u) {
    p.dZ = ws.dZ; p.ldz = ws.ldz;
    p.ztgt = ws.ztgt;
    k_gemm4w<EPI_FWDU, A_ROW, BGPO_TILE4><<<grid, kGemmThreads4, 0, s>>>(p);
  } else {
    k_gemm4w<EPI_FWD, A_ROW, BGPO_TILE4><<<grid, kGemmThreads4, 0, s>>>(p);
  }
  return hipGetLastError();
}

hipError_t launch_gemm_dx(const Workspace& ws, const uint16_t* W, int d, int V, int grid,
                          hipStream_t s) {
  // dX^T[c][row] = W[c][:] . dZ[row][:] over the unit's rows of dZ, stored
  // transposed: dx_part[row][c]
  GemmParams p = base_params();
  if (ws.Wk) {
    p.A = ws.Wk; p.lda = d;
  } else {
    p.A = W; p.lda = V;
  }
  p.B = ws.dZ; p.ldb = ws.ldz; p.dyn_boff = 1;
  p.M = d; p.K = V; p.dyn_n = 1; p.meta = ws.unit();
  p.dyn_split = 1;
  p.group_m = kGroupMdX;
  p.out = ws.dx_part; p.ldo = d; p.split_stride = ws.RP * d;
  if (ws.Wk)
    k_gemm4w<EPI_F32_STORE, A_KSLAB, BGPO_TILE4><<<grid, kGemmThreads4, 0, s>>>(p);
  else
    k_gemm4w<EPI_F32_STORE, A_ROW, BGPO_TILE4><<<grid, kGemmThreads4, 0, s>>>(p);
  return hipGetLastError();
}

hipError_t launch_gemm_dw(const Workspace& ws, float* dW, int d, int V, int grid, hipStream_t s) {
  // dW^T[v][c] += dZ[:][v] . H_c^T[c][:] over the batch's rows (dZ read
  // M-slab-major)
  GemmParams p = base_params();
  p.A = ws.dZ; p.lda = ws.ldz;
  p.B = ws.HcT; p.ldb = d;
  p.M = V; p.N = d; p.dyn_k = 1; p.meta = ws.unit();
  p.group_m = kGroupMdW;
  p.out = dW; p.ldo = V;
  k_gemm4w<EPI_F32_ACCUM, A_MSLAB, BGPO_TILE4><<<grid, kGemmThreads4, 0, s>>>(p);
  return hipGetLastError();
}

hipError_t launch_gemm_recompute(const Workspace& ws, int d, int v0, int width, int grid,
                                 hipStream_t s) {
  // Z^T[v][row] for the chunk's ids v0 .. v0 + width - 1, epilogue -> dZ
  GemmParams p = base_params();
  p.A = ws.WT + (int64_t)v0 * d; p.lda = d;
  p.B = ws.Hc; p.ldb = ws.RP;
  p.M = width; p.K = d; p.dyn_n = 1; p.meta = ws.unit();
  p.k_split = d;
  p.group_m = kGroupMFwd;
  p.lse2 = ws.lse2; p.rscale = ws.row_scale; p.rtgt = ws.row_tgt; p.v0 = v0;
  p.dZ = ws.dZ; p.ldz = ws.RP;
  k_gemm4w<EPI_DZ, A_ROW, BGPO_TILE4><<<grid, kGemmThreads4, 0, s>>>(p);
  return hipGetLastError();
}

hipError_t launch_gemm_dx_chunk(const Workspace& ws, const uint16_t* W, int d, int V, int v0,
                                int width, bool first, int grid, hipStream_t s) {
  // dX^T[c][row] (+)= W[c][v0 ..] . dZ[row][..] over the chunk, split over
  // the chunk as the unit's record says; the first chunk stores the partials
  GemmParams p = base_params();
  if (ws.Wk) {
    p.A = ws.Wk + (int64_t)v0 * d; p.lda = d;   // v0 / 64 whole slabs of d rows
  } else {
    p.A = W + v0; p.lda = V;
  }
  p.B = ws.dZ; p.ldb = ws.RP;
  p.M = d; p.K = width; p.dyn_n = 1; p.meta = ws.unit();
  p.dyn_split = 1;
  p.group_m = kGroupMdX;
  p.out = ws.dx_part; p.ldo = d; p.split_stride = ws.RP * d;
  if (ws.Wk && first)
    k_gemm4w<EPI_F32_STORE, A_KSLAB, BGPO_TILE4><<<grid, kGemmThreads4, 0, s>>>(p);
  else if (ws.Wk)
    k_gemm4w<EPI_F32_ACCUM, A_KSLAB, BGPO_TILE4><<<grid, kGemmThreads4, 0, s>>>(p);
  else if (first)
    k_gemm4w<EPI_F32_STORE, A_ROW, BGPO_TILE4><<<grid, kGemmThreads4, 0, s>>>(p);
  else
    k_gemm4w<EPI_F32_ACCUM, A_ROW, BGPO_TILE4><<<grid, kGemmThreads4, 0, s>>>(p);
  return hipGetLastError();
}

hipError_t launch_gemm_dw_chunk(const Workspace& ws, float* dW, int d, int V, int v0, int width,
                                int grid, hipStream_t s) {
  // dW^T[v0 + m][c] += dZ[:][m] . H_c^T[c][:] (K = the unit's rows; dZ read
  // M-slab-major)
  GemmParams p = base_params();
  p.A = ws.dZ; p.lda = ws.RP;
  p.B = ws.HcT; p.ldb = d;
  p.M = width; p.N = d; p.dyn_k = 1; p.meta = ws.unit();
  p.group_m = kGroupMdW;
  p.out = dW + v0; p.ldo = V;
  k_gemm4w<EPI_F32_ACCUM, A_MSLAB, BGPO_TILE4><<<grid, kGemmThreads4, 0, s>>>(p);
  return hipGetLastError();
}

int gemm_grid(int device) {
  int cus = 0;
  if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, device) != hipSuccess ||
      cus <= 0)
    cus = 256;
  return cus;  // one workgroup per compute unit
}

}  // namespace bgpo

// ---- test hook: the GEMM core alone (the dX GEMM's kernel: A slab-major, B
// row-major), C[m][n] = sum_k A[m][k] B[n][k] in fp32 ----
extern "C" int bgpo_test_gemm_nt(const uint16_t* A, const uint16_t* B, float* C, int32_t M, int32_t N,
                                 int32_t K, void* stream) {
  using namespace bgpo;
  if (!A || !B || !C || M <= 0 || N <= 0 || K <= 0 || K % 64) return -1;
  if ((int64_t)((M + 255) / 256) * ((N + 255) / 256) >= (int64_t(1) << 30)) return -1;
  // the production kernel stores C^T of its operands' product: swap them
  GemmParams p = base_params();
  p.A = B; p.lda = K; p.B = A; p.ldb = M;
  p.M = N; p.N = M; p.K = K; p.k_split = K;
  p.out = C; p.ldo = N;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return -3;
  k_gemm4w<EPI_F32_STORE, A_ROW, BGPO_TILE4><<<gemm_grid(dev), kGemmThreads4, 0, (hipStream_t)stream>>>(p);
  return hipGetLastError() == hipSuccess ? 0 : -3;
}

// ---- test hook: the GEMM core with K split into slices ----
extern "C" int bgpo_test_gemm_split(const uint16_t* A, const uint16_t* B, float* C, int32_t M,
                                    int32_t N, int32_t K, int32_t n_split, void* stream) {
  using namespace bgpo;
  if (!A || !B || !C || M <= 0 || N <= 0 || K <= 0 || K % 64 || n_split < 1 || n_split > 255)
    return -1;
  if ((int64_t)((M + 255) / 256) * ((N + 255) / 256) * n_split >= (int64_t(1) << 30)) return -1;
  // slice s covers K range [s * ks, min(K, (s + 1) * ks)) with ks a multiple
  // of 64; trailing slices can be empty (their block is stored as zeros)
  GemmParams p = base_params();
  p.A = B; p.lda = K; p.B = A; p.ldb = M;
  p.M = N; p.N = M; p.K = K;
  p.n_split = n_split;
  p.k_split = ((K + n_split - 1) / n_split + 63) / 64 * 64;
  p.out = C; p.ldo = N; p.split_stride = (int64_t)M * N;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return -3;
  k_gemm4w<EPI_F32_STORE, A_ROW, BGPO_TILE4><<<gemm_grid(dev), kGemmThreads4, 0, (hipStream_t)stream>>>(p);
  return hipGetLastError() == hipSuccess ? 0 : -3;
}

// ---- test hook: the dW GEMM's kernel alone (A M-slab-major, read through the
// transposing LDS reads; B K-slab-major), C[n][m] += sum_k A[m][k] B[n][k] ----
extern "C" int bgpo_test_gemm_tn(const uint16_t* A, const uint16_t* B, float* C, int32_t M, int32_t N,
                                 int32_t K, void* stream) {
  using namespace bgpo;
  if (!A || !B || !C || M <= 0 || N <= 0 || K <= 0 || K % 64 || M % 64) return -1;
  if ((int64_t)((M + 255) / 256) * ((N + 255) / 256) >= (int64_t(1) << 30)) return -1;
  GemmParams p = base_params();
  p.A = A; p.lda = K;          // [M/64][K][64]
  p.B = B; p.ldb = N;          // [K/64][N][64]
  p.M = M; p.N = N; p.K = K;
  p.group_m = kGroupMdW;
  p.out = C; p.ldo = M;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return -3;
  k_gemm4w<EPI_F32_ACCUM, A_MSLAB, BGPO_TILE4><<<gemm_grid(dev), kGemmThreads4, 0, (hipStream_t)stream>>>(p);
  return hipGetLastError() == hipSuccess ? 0 : -3;
}
