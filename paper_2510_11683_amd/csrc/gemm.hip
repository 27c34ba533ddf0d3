// bf16 MFMA GEMM cores for gfx950 and their four epilogues.
//
// Every contraction of the ELBO head is written in one "NT" form,
//     C[m][n] = sum_k A[m][k] * B[n][k]      (A, B row-major, K contiguous),
// so both operands load as 16-byte K-contiguous vectors that match the MFMA
// operand layouts directly:
//   forward               Z^T[v][row] = WT[v][:] . Hc[row][:]     (K = d)
//   dX (split over V)     dX^T[c][row] = W[c][:] . dZ[row][:]     (K = V)
//   dW                    dW^T[v][c]  += dZT[v][:] . HcT[c][:]    (K = rows)
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
// k_gemm4w (production): four waves of 128x128 on 16x16x32 MFMAs in inline
// assembly with accumulators in AGPRs, hand-ordered (see below).  k_gemm
// (the earlier core, kept for the tile-configuration test hook): eight waves
// of 128x64 on compiler-scheduled 32x32x16 MFMAs.
#include "common.hpp"
#include "internal.hpp"

#include <string.h>

namespace bgpo {

enum EpiKind { EPI_FWD = 0, EPI_FWDU = 1, EPI_F32_STORE = 2, EPI_F32_ACCUM = 3 };

struct GemmParams {
  const uint16_t* A;
  int64_t lda;
  const uint16_t* B;
  int64_t ldb;
  int M, N, K;               // static extents
  int dyn_m, dyn_n, dyn_k;   // extents taken from the device sample metadata
  int dyn_split;             // K split taken from the metadata (dX)
  int n_split;               // K split count
  int64_t k_split;           // K per split (multiple of BK)
  int group_m;              // tile order: bands of group_m M tiles, walking along N
                             // (1 = N tiles consecutive, tilesM = M tiles consecutive)
  int plain_order;           // 1 = no XCD grouping of consecutive tiles (experiments)
  const SampleMeta* meta;
  // epilogue operands
  float* out;                // F32 store / accumulate target
  int64_t ldo, split_stride;
  float* part_m;             // FWD: per-128-vocabulary-slice (max, sum) partials [M/WM][ldp]
  float* part_s;
  int64_t ldp;
  uint16_t* dZ;              // FWDU: exponentials u, [rows][ldz]
  int64_t ldz;
};

template <int BM, int BN, int BK, int WM, int WN, int SWZ = 0>
struct Cfg {
  static constexpr int NWM = BM / WM, NWN = BN / WN;
  static constexpr int NWAVES = NWM * NWN;
  static constexpr int NT = NWAVES * 64;
  static constexpr int TM = WM / 32, TN = WN / 32;
  static constexpr int KCH = BK / 8;                  // 16-byte chunks per LDS row
  static constexpr int A_LD = BM * KCH / NT, B_LD = BN * KCH / NT;
  static constexpr int ROWS_PER_128B = 8 / KCH;
  static_assert(BM * KCH % NT == 0 && BN * KCH % NT == 0, "load split");
  static_assert(KCH == 4 || KCH == 8, "BK must be 32 or 64");
  // 16-byte chunk c of LDS row r is stored at chunk c ^ swz(r).  SWZ 0 makes 8
  // consecutive rows hit 8 distinct 16-byte slots of a 128-byte bank line;
  // SWZ 1 spreads 16 consecutive rows over 256 bytes (pairs of rows share a
  // key, and consecutive rows already alternate 128-byte halves).
  __device__ static __forceinline__ int swz(int row) {
    return SWZ == 0 ? (row / ROWS_PER_128B) % KCH : ((row >> 1) / ROWS_PER_128B) % KCH;
  }
};

// fp32 store of a wave tile (ACCUM: read-modify-write), one 32-row band at a
// time so the loads stay in flight without spills.
template <bool ACCUM, bool FULL, int TM, int TN>
__device__ __forceinline__ void epi_f32(const f32x16 (&acc)[TM][TN], float* outb, int64_t ldo,
                                        int mw, int nw, int mlane, int lane, int M, int N) {
#pragma unroll
  for (int i = 0; i < TM; ++i) {
    float old[TN][16];
    if constexpr (ACCUM) {
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const int n = nw + 32 * j + (lane & 31);
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int m = mw + 32 * i + mlane + (e & 3) + 8 * (e >> 2);
          old[j][e] = (FULL || (m < M && n < N)) ? outb[(int64_t)m * ldo + n] : 0.f;
        }
      }
    }
#pragma unroll
    for (int j = 0; j < TN; ++j) {
      const int n = nw + 32 * j + (lane & 31);
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int m = mw + 32 * i + mlane + (e & 3) + 8 * (e >> 2);
        if (FULL || (m < M && n < N))
          outb[(int64_t)m * ldo + n] = ACCUM ? old[j][e] + acc[i][j][e] : acc[i][j][e];
      }
    }
    __builtin_amdgcn_sched_barrier(0);
  }
}

// Issue one K slab of both operand tiles into LDS stage `stage`.
// s_waitcnt vmcnt(N) with the other counters left alone (gfx9 encoding: vmcnt
// in bits 3:0 and 15:14, expcnt 6:4, lgkmcnt 11:8).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// MFMA operand fragments of K sub-step ks of LDS stage `stage`: lane l holds the
// 8 consecutive K values 8 (2 ks + l / 32) .. +7 of row l % 32 of each 32-row
// band of the wave's A and B sub-tiles.
template <int BM, int BN, int KCH, int TM, int TN, int WM, int WN, class C>
__device__ __forceinline__ void read_frags(bf16x8 (&fa)[TM], bf16x8 (&fb)[TN], const uint4* As,
                                           const uint4* Bs, int stage, int ks, int wm, int wn,
                                           int lane) {
  const int ch = ks * 2 + (lane >> 5);
  const uint4* Ac = As + stage * BM * KCH;
  const uint4* Bc = Bs + stage * BN * KCH;
  // issue order = order of first use by the next sub-step's MFMAs (i outer,
  // j inner): B0, A0, B1, A1, then the remaining fragments
  auto ra = [&](int i) {
    const int row = wm * WM + i * 32 + (lane & 31);
    fa[i] = __builtin_bit_cast(bf16x8, Ac[row * KCH + (ch ^ C::swz(row))]);
  };
  auto rb = [&](int j) {
    const int row = wn * WN + j * 32 + (lane & 31);
    fb[j] = __builtin_bit_cast(bf16x8, Bc[row * KCH + (ch ^ C::swz(row))]);
  };
#pragma unroll
  for (int q = 0; q < (TM > TN ? TM : TN); ++q) {
    if (q < TN) rb(q);
    if (q < TM) ra(q);
  }
}

template <int BM, int BN, int KCH, int A_INS, int B_INS, int STAGES>
__device__ __forceinline__ void issue_slab_loads(uint4* As, uint4* Bs, int stage, int wave,
                                                 __amdgpu_buffer_rsrc_t a_rsrc,
                                                 __amdgpu_buffer_rsrc_t b_rsrc,
                                                 const uint32_t (&a_voff)[A_INS],
                                                 const uint32_t (&b_voff)[B_INS], int soff) {
#if defined(__HIP_DEVICE_COMPILE__)
#pragma unroll
  for (int q = 0; q < A_INS; ++q) {
    uint4* dst = As + stage * BM * KCH + (wave * A_INS + q) * 64;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(
        a_rsrc, (__attribute__((address_space(3))) void*)dst, 16, a_voff[q], soff, 0, 0);
  }
#pragma unroll
  for (int q = 0; q < B_INS; ++q) {
    uint4* dst = Bs + stage * BN * KCH + (wave * B_INS + q) * 64;
    __builtin_amdgcn_raw_ptr_buffer_load_lds(
        b_rsrc, (__attribute__((address_space(3))) void*)dst, 16, b_voff[q], soff, 0, 0);
  }
#endif
}

// Instruction-order template for one K sub-step: MF MFMAs with ND LDS
// fragment reads and NV slab loads placed between them (one scheduling group
// per instruction kind and position; requires ND <= MF).
template <int I, int MF, int NV, int ND>
__device__ __forceinline__ void sched_pattern() {
#if defined(__HIP_DEVICE_COMPILE__)
  if constexpr (I < MF) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);            // MFMA
    // fragment reads and slab loads both spread evenly over the step's MFMA
    // slots (measured: front-loading the reads made no difference for the
    // forward and cost 2-3 % of MFMA-busy cycles in the dX and dW GEMMs)
    constexpr int v = (I + 1) * NV / MF - I * NV / MF;
    constexpr int d = (I + 1) * ND / MF - I * ND / MF;
    if constexpr (d > 0) __builtin_amdgcn_sched_group_barrier(0x100, d, 0);   // DS read
    if constexpr (v > 0) __builtin_amdgcn_sched_group_barrier(0x020, v, 0);   // VMEM read
    sched_pattern<I + 1, MF, NV, ND>();
  }
#endif
}

template <int EPI, int BM, int BN, int BK, int WM, int WN, int STAGES, int OCC = 1, int SWZ = 0>
__global__ __launch_bounds__((BM / WM) * (BN / WN) * 64, OCC) void k_gemm(GemmParams p) {
#if defined(__HIP_DEVICE_COMPILE__)  // the host pass needs only the signature
  using C = Cfg<BM, BN, BK, WM, WN, SWZ>;
  constexpr int NT = C::NT, TM = C::TM, TN = C::TN, KCH = C::KCH, KS = BK / 16;
  __shared__ uint4 smem[STAGES * (BM + BN) * KCH];
  uint4* As = smem;                           // [STAGES][BM][KCH]
  uint4* Bs = smem + STAGES * BM * KCH;       // [STAGES][BN][KCH]

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave-uniform, kept in an SGPR
  const int wm = wave / C::NWN, wn = wave % C::NWN;

  int M = p.M, N = p.N, K = p.K, n_valid = p.N;
  if (p.dyn_m) { M = p.meta->n_rows_pad; n_valid = p.meta->n_rows; }
  if (p.dyn_n) { N = p.meta->n_rows_pad; n_valid = p.meta->n_rows; }
  if (p.dyn_k) K = p.meta->col_end;    // batched dW: all samples' columns (multiple of 64)
  int n_split = p.n_split;
  int64_t k_split = p.k_split;
  if (p.dyn_split) {
    n_split = p.meta->dx_split;
    k_split = (int64_t)p.meta->dx_kslab * BK;
  }
  if (EPI == EPI_F32_ACCUM && K == 0) return;   // nothing to add
  const int tilesM = (M + BM - 1) / BM, tilesN = (N + BN - 1) / BN;
  const int64_t total = (int64_t)tilesM * tilesN * n_split;
  const int G = gridDim.x;
  const int w = blockIdx.x;
  const int xcd_slot = (G % 8 == 0 && !p.plain_order) ? (w % 8) * (G / 8) + w / 8 : w;

  for (int64_t base = 0; base < total; base += G) {
    const int64_t t = base + xcd_slot;
    if (t >= total) continue;
    int mt, nt, split;
    {
      // bands of GM M tiles walk along N, so a run of consecutive tiles (the
      // ones an XCD holds at once) covers about GM x (run / GM) tiles and
      // touches GM + run / GM operand panels
      const int64_t per_split = (int64_t)tilesM * tilesN;
      split = (int)(t / per_split);
      const int64_t r = t - (int64_t)split * per_split;
      const int GM = max(1, min(p.group_m, tilesM));
      const int64_t band = r / ((int64_t)GM * tilesN);
      const int gm = min(GM, tilesM - (int)band * GM);   // the last band may be shorter
      const int64_t idx = r - band * GM * tilesN;
      mt = (int)band * GM + (int)(idx % gm);
      nt = (int)(idx / gm);
    }
    const int m0 = mt * BM, n0 = nt * BN;
    const int64_t kb = (int64_t)split * k_split;
    const int64_t ke = min((int64_t)K, kb + k_split);
    const int nk = ke > kb ? (int)((ke - kb) / BK) : 0;

    // accumulator element (i, j, e) sits at
    //   m = mw + 32 i + 4 (lane >> 5) + (e & 3) + 8 (e >> 2),  n = nw + 32 j + (lane & 31)
    const int mw = m0 + wm * WM, nw = n0 + wn * WN;
    const int mlane = 4 * (lane >> 5);
    f32x16 acc[TM][TN];
    // dW accumulates in place: a full tile starts from the current output
    // (buffer loads issued before the slab loads, so the wait for the first
    // slab covers them) and ends with plain stores; a partial tile starts
    // from zero and adds in its epilogue
    const bool preload = EPI == EPI_F32_ACCUM && m0 + BM <= M && n0 + BN <= N;
    if (preload) {
      const float* src = p.out + (int64_t)split * p.split_stride + (int64_t)m0 * p.ldo + n0;
      const __amdgpu_buffer_rsrc_t o_rsrc =
          __builtin_amdgcn_make_buffer_rsrc((void*)src, (short)0, 0x7FFFFFFF, 0x00020000);
      const int lane_off = ((mw - m0 + mlane) * (int)p.ldo + (nw - n0) + (lane & 31)) * 4;
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
          for (int e = 0; e < 16; ++e)
            acc[i][j][e] = __builtin_bit_cast(
                float, __builtin_amdgcn_raw_buffer_load_b32(
                           o_rsrc, lane_off,
                           ((32 * i + (e & 3) + 8 * (e >> 2)) * (int)p.ldo + 32 * j) * 4, 0));
    } else {
#pragma unroll
      for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
          for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;
    }

    // Operand panels as buffer resources (wave-uniform): rows [m0, m0 + BM) of A
    // and [n0, n0 + BN) of B.  Each load instruction moves 64 lanes x 16 bytes
    // straight into LDS (lane l lands at byte 16 l of the instruction's LDS
    // block), so the XOR swizzle is applied on the global side: lane l of
    // block g fetches logical chunk (l mod KCH) ^ swz(row) of row
    // g * RPI + l / KCH.  Rows past the matrix are clamped to its last row.
    const __amdgpu_buffer_rsrc_t a_rsrc = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(p.A + (int64_t)m0 * p.lda), (short)0, 0x7FFFFFFF, 0x00020000);
    const __amdgpu_buffer_rsrc_t b_rsrc = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(p.B + (int64_t)n0 * p.ldb), (short)0, 0x7FFFFFFF, 0x00020000);
    constexpr int RPI = 64 / KCH;                        // rows per load instruction
    constexpr int A_INS = BM / RPI / C::NWAVES, B_INS = BN / RPI / C::NWAVES;
    uint32_t a_voff[A_INS], b_voff[B_INS];
#pragma unroll
    for (int q = 0; q < A_INS; ++q) {
      const int g = wave * A_INS + q, row = g * RPI + lane / KCH;
      const int c = (lane % KCH) ^ C::swz(row);
      const int rr = min(m0 + row, M - 1) - m0;
      a_voff[q] = (uint32_t)(rr * p.lda * 2 + c * 16);
    }
#pragma unroll
    for (int q = 0; q < B_INS; ++q) {
      const int g = wave * B_INS + q, row = g * RPI + lane / KCH;
      const int c = (lane % KCH) ^ C::swz(row);
      const int rr = min(n0 + row, N - 1) - n0;
      b_voff[q] = (uint32_t)(rr * p.ldb * 2 + c * 16);
    }
    if (nk > 0) {
      // S-stage ring of K slabs: slab q lives in stage q % S.  The prologue
      // fills all S stages; at the barrier that ends slab c every wave has
      // read all of slab c's stage, so slab c + S is loaded into it right
      // away and has S - 1 slabs of MFMA time to land.  Slabs past the end of
      // this tile's K range re-load its last slab into a stage no later slab
      // uses, so every wave always has the same number of load groups in
      // flight and the vmcnt waits are compile-time constants.
      constexpr int NINS = A_INS + B_INS;
      constexpr int NFRAG = TM + TN;
      auto issue = [&](int q) {
        const int qc = min(q, nk - 1);
        issue_slab_loads<BM, BN, KCH, A_INS, B_INS, STAGES>(As, Bs, q % STAGES, wave, a_rsrc,
                                                            b_rsrc, a_voff, b_voff,
                                                            (int)((kb + (int64_t)qc * BK) * 2));
      };
#pragma unroll
      for (int q = 0; q < STAGES; ++q) issue(q);
      wait_vmcnt<NINS * (STAGES - 1)>();
      __builtin_amdgcn_s_barrier();

      bf16x8 fa[2][TM], fb[2][TN];
      auto mfma_step = [&](int h) {
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int j = 0; j < TN; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[h][i], fb[h][j], acc[i][j], 0, 0, 0);
      };
      read_frags<BM, BN, KCH, TM, TN, WM, WN, C>(fa[0], fb[0], As, Bs, 0, 0, wm, wn, lane);
      for (int kt = 0; kt + 1 < nk; ++kt) {
        const int cur = kt % STAGES;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          if (ks + 1 < KS) {
            read_frags<BM, BN, KCH, TM, TN, WM, WN, C>(fa[(ks + 1) & 1], fb[(ks + 1) & 1], As, Bs,
                                                        cur, ks + 1, wm, wn, lane);
            mfma_step(ks & 1);
            sched_pattern<0, TM * TN, 0, NFRAG>();
          } else {
            // slab kt+1 landed (own loads) and, after the barrier, every wave
            // has finished reading stage `cur`: refill it with slab kt+S while
            // the last MFMAs of slab kt run, and start reading slab kt+1.
            wait_vmcnt<NINS * (STAGES - 2)>();
            __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0)
            __builtin_amdgcn_s_barrier();
            __builtin_amdgcn_sched_barrier(0);
            issue(kt + STAGES);
            read_frags<BM, BN, KCH, TM, TN, WM, WN, C>(fa[(ks + 1) & 1], fb[(ks + 1) & 1], As, Bs,
                                                        (kt + 1) % STAGES, 0, wm, wn, lane);
            mfma_step(ks & 1);
            sched_pattern<0, TM * TN, NINS, NFRAG>();
          }
          __builtin_amdgcn_sched_barrier(0);
        }
      }
      // the last slab
      {
        const int cur = (nk - 1) % STAGES;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
          if (ks + 1 < KS) {
            read_frags<BM, BN, KCH, TM, TN, WM, WN, C>(fa[(ks + 1) & 1], fb[(ks + 1) & 1], As, Bs,
                                                        cur, ks + 1, wm, wn, lane);
            mfma_step(ks & 1);
            sched_pattern<0, TM * TN, 0, NFRAG>();
          } else {
            mfma_step(ks & 1);
          }
          __builtin_amdgcn_sched_barrier(0);
        }
      }
      // drain the ring (outstanding re-loads) before the epilogue may reuse LDS
      __builtin_amdgcn_s_waitcnt(0);
      __builtin_amdgcn_s_barrier();
    }

    // ---------------- epilogues ----------------
    if constexpr (EPI == EPI_FWD || EPI == EPI_FWDU) {
      // Per (row, 128-entry vocabulary slice of this wave): max m and sum of
      // 2^(z log2e - m), in log2 units, written straight to the partials (the
      // slice of wave row wm is partial index mw / 128).  Lanes l and l ^ 32
      // hold the two halves of a row's slice.  EPI_FWDU also stores the
      // exponentials u = 2^(z log2e - m) as fp16 into dZ[row][v] (each lane
      // holds 4 consecutive vocabulary ids of a row: 8-byte stores); the
      // softmax-gradient kernel later turns them into s (p - onehot) with
      // p = u 2^(m - lse) and writes the transposed copy.  Both variants sum
      // in the same order, so l is bit-identical between them.  No LDS is
      // used here.
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
            for (int e = 0; e < 16; ++e)
              if (mw + 32 * i + mlane + (e & 3) + 8 * (e >> 2) >= M) acc[i][j][e] = -INFINITY;
      }
      // EPI_FWDU stages the tile's exponentials in LDS (free once the ring is
      // drained; 256 rows x 256 vocabulary ids x fp16 = the ring's 128 KB) as
      // [row][vocabulary], 16-byte chunk c of row r at chunk c ^ (r mod 32) so
      // that the 32 rows one write instruction touches hit distinct banks; the
      // rows are then written out whole (two 512-byte rows per instruction)
      // instead of 8-byte pieces scattered over 32 rows.
      char* stage_u = reinterpret_cast<char*>(smem);
      static_assert(!kStore || (BM == 256 && BN == 256 && STAGES * (BM + BN) * KCH * 16 >= BM * BN * 2),
                    "staging tile: 512-byte rows that fit the ring");
      float mref[TN], ssum[TN];
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        float mx = -INFINITY;
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int e = 0; e < 16; ++e) mx = fmaxf(mx, acc[i][j][e]);
        mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
        mref[j] = mx > -INFINITY ? mx * kLog2e : 0.f;        // a slice past V has no entries
        ssum[j] = 0.f;
      }
#pragma unroll
      for (int i = 0; i < TM; ++i) {
#pragma unroll
        for (int j = 0; j < TN; ++j) {
          const int n = nw + 32 * j + (lane & 31);
          uint32_t pk[8];   // pk[q] = (id 2q, id 2q+1) of this lane's row
#pragma unroll
          for (int q = 0; q < 8; ++q) {
            const float u0 = __builtin_amdgcn_exp2f(fmaf(acc[i][j][2 * q], kLog2e, -mref[j]));
            const float u1 = __builtin_amdgcn_exp2f(fmaf(acc[i][j][2 * q + 1], kLog2e, -mref[j]));
            ssum[j] += u0 + u1;
            if constexpr (kStore) pk[q] = pack_f16x2(u0, u1);
          }
          if constexpr (kStore) {
            // into the LDS staging tile: vocabulary ids m .. m+3 of row n
            const int nl = n - n0;
#pragma unroll
            for (int e4 = 0; e4 < 4; ++e4) {
              const int ml = mw - m0 + 32 * i + 8 * e4;
              *reinterpret_cast<uint2*>(stage_u + nl * 512 + (((ml >> 3) ^ (nl & 31)) << 4) +
                                        mlane * 2) = make_uint2(pk[2 * e4], pk[2 * e4 + 1]);
            }
          }
        }
      }
      const int vt = mw / WM;
#pragma unroll
      for (int j = 0; j < TN; ++j) {
        const float st = ssum[j] + __shfl_xor(ssum[j], 32, 64);
        const int n = nw + 32 * j + lane;
        if (lane < 32 && mw < M && n < n_valid) {
          p.part_m[(int64_t)vt * p.ldp + n] = mref[j];
          p.part_s[(int64_t)vt * p.ldp + n] = st;
        }
      }
      if constexpr (kStore) {
        __syncthreads();
        // lane l of a store instruction: row 2 q + l / 32 of the wave's rows,
        // stored chunk l mod 32, i.e. logical chunk (l mod 32) ^ (row mod 32)
        constexpr int ROWS_PER_WAVE = BN / (NT / 64);
        // (the lane's chunk is re-derived here every tile: hoisted out of the
        // tile loop, its 16 per-row variants would be spilled)
        int pc = lane & 31;
        asm volatile("" : "+v"(pc));
#pragma unroll
        for (int q = 0; q < ROWS_PER_WAVE / 2; ++q) {
          const int row = wave * ROWS_PER_WAVE + 2 * q + (lane >> 5);
          const int m = m0 + 8 * (pc ^ (row & 31));
          const uint4 v = *reinterpret_cast<const uint4*>(stage_u + row * 512 + pc * 16);
          if (n0 + row < N && m < M)
            *reinterpret_cast<uint4*>(p.dZ + (int64_t)(n0 + row) * p.ldz + m) = v;
        }
      }
    } else {
      // fp32 store of the tile (dX partials, or a full dW tile that started
      // from its previous value), or read-modify-write of a partial dW tile;
      // one 32-row band of the wave tile at a time.
      float* outb = p.out + (int64_t)split * p.split_stride;
      if (m0 + BM <= M && n0 + BN <= N) epi_f32<false, true, TM, TN>(acc, outb, p.ldo, mw, nw, mlane, lane, M, N);
      else epi_f32<EPI == EPI_F32_ACCUM, false, TM, TN>(acc, outb, p.ldo, mw, nw, mlane, lane, M, N);
    }
    __syncthreads();
  }
#endif
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

template <int EPI, int BM, int BN, int BK, int STAGES, int SWZ>
__global__ __launch_bounds__(256, 1) void k_gemm4w(GemmParams p) {
#if defined(__HIP_DEVICE_COMPILE__)  // the host pass needs only the signature
  constexpr int WM = 128, WN = 128;
  using C = Cfg<BM, BN, BK, WM, WN, SWZ>;
  constexpr int NT = C::NT, KCH = C::KCH;
  constexpr int TM = WM / 16, TN = WN / 16;
  // 64-deep slabs hold two 32-deep MFMA sub-steps between barriers; 32-deep
  // slabs one, so a ring of the same LDS size has twice the stages
  static_assert(C::NWAVES == 4 && (BK == 64 || BK == 32), "four waves, 32- or 64-deep slabs");
  __shared__ uint4 smem[STAGES * (BM + BN) * KCH];
  uint4* As = smem;                           // [STAGES][BM][KCH]
  uint4* Bs = smem + STAGES * BM * KCH;       // [STAGES][BN][KCH]

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave-uniform, kept in an SGPR
  const int wm = wave / C::NWN, wn = wave % C::NWN;

  int M = p.M, N = p.N, K = p.K, n_valid = p.N;
  if (p.dyn_m) { M = p.meta->n_rows_pad; n_valid = p.meta->n_rows; }
  if (p.dyn_n) { N = p.meta->n_rows_pad; n_valid = p.meta->n_rows; }
  if (p.dyn_k) K = p.meta->col_end;    // batched dW: all samples' columns (multiple of 64)
  int n_split = p.n_split;
  int64_t k_split = p.k_split;
  if (p.dyn_split) {
    n_split = p.meta->dx_split;
    k_split = (int64_t)p.meta->dx_kslab * 64;   // 64-wide slabs: nk even for BK 32
  }
  if (EPI == EPI_F32_ACCUM && K == 0) return;   // nothing to add
  const int tilesM = (M + BM - 1) / BM, tilesN = (N + BN - 1) / BN;
  const int64_t total = (int64_t)tilesM * tilesN * n_split;
  const int G = gridDim.x;
  const int w = blockIdx.x;
  const int xcd_slot = (G % 8 == 0 && !p.plain_order) ? (w % 8) * (G / 8) + w / 8 : w;

  for (int64_t base = 0; base < total; base += G) {
    const int64_t t = base + xcd_slot;
    if (t >= total) continue;
    // the lane index, re-derived every tile: addresses computed from it are
    // then not hoisted out of the tile loop (with all 256 AGPRs holding
    // accumulators, such hoisted values would be spilled)
    int lane_t = tid & 63;
    asm volatile("" : "+v"(lane_t));
    const int lane = lane_t;
    int mt, nt, split;
    {
      // bands of GM M tiles walk along N (as in k_gemm)
      const int64_t per_split = (int64_t)tilesM * tilesN;
      split = (int)(t / per_split);
      const int64_t r = t - (int64_t)split * per_split;
      const int GM = max(1, min(p.group_m, tilesM));
      const int64_t band = r / ((int64_t)GM * tilesN);
      const int gm = min(GM, tilesM - (int)band * GM);
      const int64_t idx = r - band * GM * tilesN;
      mt = (int)band * GM + (int)(idx % gm);
      nt = (int)(idx / gm);
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
    // global side; rows past the matrix are clamped to its last row.
    const __amdgpu_buffer_rsrc_t a_rsrc = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(p.A + (int64_t)m0 * p.lda), (short)0, 0x7FFFFFFF, 0x00020000);
    const __amdgpu_buffer_rsrc_t b_rsrc = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(p.B + (int64_t)n0 * p.ldb), (short)0, 0x7FFFFFFF, 0x00020000);
    constexpr int RPI = 64 / KCH;                        // rows per load instruction
    constexpr int A_INS = BM / RPI / C::NWAVES, B_INS = BN / RPI / C::NWAVES;
    static_assert(A_INS + B_INS == BK / 4, "one slab load per 256 / BK MFMAs");
    uint32_t a_voff[A_INS], b_voff[B_INS];
#pragma unroll
    for (int q = 0; q < A_INS; ++q) {
      const int g = wave * A_INS + q, row = g * RPI + lane / KCH;
      const int c = (lane % KCH) ^ C::swz(row);
      const int rr = min(m0 + row, M - 1) - m0;
      a_voff[q] = (uint32_t)(rr * p.lda * 2 + c * 16);
    }
#pragma unroll
    for (int q = 0; q < B_INS; ++q) {
      const int g = wave * B_INS + q, row = g * RPI + lane / KCH;
      const int c = (lane % KCH) ^ C::swz(row);
      const int rr = min(n0 + row, N - 1) - n0;
      b_voff[q] = (uint32_t)(rr * p.ldb * 2 + c * 16);
    }
    if (nk > 0) {
      // S-stage ring of K slabs as in k_gemm: slab q lives in stage q % S,
      // slab c + S is loaded into slab c's stage right after the barrier that
      // ends slab c, and slabs past the tile's K range re-load its last slab.
      constexpr int NINS = A_INS + B_INS;
      auto issue_one = [&](int q, int stage, int e) {   // load instruction e of slab q
        const int qc = min(q, nk - 1);
        const int soff = (int)((kb + (int64_t)qc * BK) * 2);
        if (e < A_INS) {
          uint4* dst = As + stage * BM * KCH + (wave * A_INS + e) * 64;
          __builtin_amdgcn_raw_ptr_buffer_load_lds(
              a_rsrc, (__attribute__((address_space(3))) void*)dst, 16, a_voff[e], soff, 0, 0);
        } else {
          uint4* dst = Bs + stage * BN * KCH + (wave * B_INS + e - A_INS) * 64;
          __builtin_amdgcn_raw_ptr_buffer_load_lds(
              b_rsrc, (__attribute__((address_space(3))) void*)dst, 16, b_voff[e - A_INS], soff,
              0, 0);
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
        } else {
          const int row = arow + 16 * (r - TN);
          da[r - TN] =
              __builtin_bit_cast(bf16x8, As[st * BM * KCH + row * KCH + (ch ^ C::swz(row))]);
        }
      };
      // one sub-step on fragment set h: its 64 MFMAs, the reads of sub-step
      // (nst, nks) into set 1 - h and, with `loads`, slab lq into stage lst
      constexpr int LEVERY = TM * TN / NINS;   // MFMAs per slab load
      auto step = [&](int h, int nst, int nks, bool loads, int lq, int lst) {
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
          for (int j = 0; j < TN; ++j) {
            const int m = i * TN + j;
            BGPO_MFMA16(acc[i][j], fa[h][i], fb[h][j]);
            if (loads && m % LEVERY == 1) issue_one(lq, lst, m / LEVERY);
            if ((m & 3) == 3) rd(fa[1 - h], fb[1 - h], nst, nks, m >> 2);
            __builtin_amdgcn_sched_barrier(0);
          }
      };
#pragma unroll
      for (int r = 0; r < TM + TN; ++r) rd(fa[0], fb[0], 0, 0, r);
      // every slab, the last one included, runs the same code (the last
      // one's reads and loads fetch data nobody uses), so the accumulators
      // stay in their registers across the whole loop
      if constexpr (BK == 64) {
        for (int kt = 0; kt < nk; ++kt) {
          const int cur = kt % STAGES;
          step(0, cur, 1, false, 0, 0);
          // slab kt + 1 landed (own loads) and, after the barrier, every wave
          // is done with stage `cur`: refill it with slab kt + S during the
          // second sub-step, which also reads slab kt + 1's first fragments
          wait_vmcnt<NINS * (STAGES - 2)>();
          __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0)
          __builtin_amdgcn_s_barrier();
          __builtin_amdgcn_sched_barrier(0);
          step(1, (kt + 1) % STAGES, 0, true, kt + STAGES, cur);
        }
      } else {
        // one sub-step per slab; K ranges are multiples of 64, so nk is even
        // and the fragment sets alternate in a fixed order.  Before slab s:
        // slab s + 1 landed, every wave is done reading stage s % S (its
        // fragments were read during slab s - 1), so slab s + S refills it
        // and has S - 1 sub-steps to land
        auto sub = [&](int h, int s) {
          wait_vmcnt<NINS * (STAGES - 2)>();
          __builtin_amdgcn_s_waitcnt(0xC07F);   // lgkmcnt(0)
          __builtin_amdgcn_s_barrier();
          __builtin_amdgcn_sched_barrier(0);
          step(h, (s + 1) % STAGES, 0, true, s + STAGES, s % STAGES);
        };
        for (int kt = 0; kt < nk; kt += 2) {
          sub(0, kt);
          sub(1, kt + 1);
        }
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
      // the exponentials u = 2^(z log2e - m) as fp16 in dZ[row][v]; the
      // softmax-gradient kernel turns them into s (p - onehot) with
      // p = u 2^(m - lse).  Both variants sum in the same order, so l is
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
      // EPI_FWDU stages the tile's exponentials in LDS (free once the ring is
      // drained; 256 rows x 256 vocabulary ids x fp16 = the ring's 128 KB) as
      // [row][vocabulary], 16-byte chunk c of row r at chunk c ^ (r mod 32),
      // and then writes whole rows (two 512-byte rows per instruction).
      char* stage_u = reinterpret_cast<char*>(smem);
      static_assert(!kStore || (BM == 256 && BN == 256 && STAGES * (BM + BN) * KCH * 16 >= BM * BN * 2),
                    "staging tile: 512-byte rows that fit the ring");
      // one 16-row column block of the wave tile at a time, so that only its
      // 32 values per lane are live outside the accumulators
      const int vt = mw / WM;
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
#pragma unroll
        for (int i = 0; i < TM; ++i) {
          float u[4];
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            u[e] = __builtin_amdgcn_exp2f(fmaf(acc[i][j][e], kLog2e, -mref));
            ssum += u[e];
          }
          if constexpr (kStore) {
            // vocabulary ids ml .. ml + 3 of row nl into the staging tile
            const int ml = mw - m0 + 16 * i + mlane;
            *reinterpret_cast<uint2*>(stage_u + nl * 512 + (((ml >> 3) ^ (nl & 31)) << 4) +
                                      (ml & 7) * 2) =
                make_uint2(pack_f16x2(u[0], u[1]), pack_f16x2(u[2], u[3]));
          }
        }
        float st = ssum + __shfl_xor(ssum, 16, 64);
        st += __shfl_xor(st, 32, 64);
        const int n = n0 + nl;
        if (lane < 16 && mw < M && n < n_valid) {
          p.part_m[(int64_t)vt * p.ldp + n] = mref;
          p.part_s[(int64_t)vt * p.ldp + n] = st;
        }
        __builtin_amdgcn_sched_barrier(0);
      }
      if constexpr (kStore) {
        __syncthreads();
        // lane l of a store instruction: row 2 q + l / 32 of the wave's rows,
        // stored chunk l mod 32, i.e. logical chunk (l mod 32) ^ (row mod 32)
        constexpr int ROWS_PER_WAVE = BN / (NT / 64);
        // (the lane's chunk is re-derived here every tile: hoisted out of the
        // tile loop, its per-row variants would be spilled)
        int pc = lane & 31;
        asm volatile("" : "+v"(pc));
#pragma unroll
        for (int q = 0; q < ROWS_PER_WAVE / 2; ++q) {
          const int row = wave * ROWS_PER_WAVE + 2 * q + (lane >> 5);
          const int m = m0 + 8 * (pc ^ (row & 31));
          const uint4 v = *reinterpret_cast<const uint4*>(stage_u + row * 512 + pc * 16);
          if (n0 + row < N && m < M)
            *reinterpret_cast<uint4*>(p.dZ + (int64_t)(n0 + row) * p.ldz + m) = v;
        }
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
// swizzle.  The eight-wave k_gemm configuration they replaced is test hook
// variant 8.
#define BGPO_TILE4 256, 256, 64, 2, 1
constexpr int kGemmThreads4 = 256;
// band heights of the tile walk (see the tile-order comment in k_gemm),
// measured at the LLaDA head shape: dW and dX fastest with bands of 8, the
// forward GEMM insensitive between 1 and 8
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
  p.B = ws.Hc; p.ldb = d;
  p.M = V; p.K = d; p.dyn_n = 1; p.meta = ws.unit();
  p.k_split = d;
  p.part_m = ws.part_m; p.part_s = ws.part_s; p.ldp = ws.RP;
  p.group_m = kGroupMFwd;
  if (store_u) {
    p.dZ = ws.dZ; p.ldz = V;
    k_gemm4w<EPI_FWDU, BGPO_TILE4><<<grid, kGemmThreads4, 0, s>>>(p);
  } else {
    k_gemm4w<EPI_FWD, BGPO_TILE4><<<grid, kGemmThreads4, 0, s>>>(p);
  }
  return hipGetLastError();
}

hipError_t launch_gemm_dx(const Workspace& ws, const uint16_t* W, int d, int V, int grid,
                          hipStream_t s) {
  // dX^T[c][row] = W[c][:] . dZ[row][:], stored transposed: dx_part[row][c]
  GemmParams p = base_params();
  p.A = W; p.lda = V;
  p.B = ws.dZ; p.ldb = V;
  p.M = d; p.K = V; p.dyn_n = 1; p.meta = ws.unit();
  p.dyn_split = 1;
  p.group_m = kGroupMdX;
  p.out = ws.dx_part; p.ldo = d; p.split_stride = ws.RP * d;
  k_gemm4w<EPI_F32_STORE, BGPO_TILE4><<<grid, kGemmThreads4, 0, s>>>(p);
  return hipGetLastError();
}

hipError_t launch_gemm_dw(const Workspace& ws, float* dW, int d, int V, int grid, hipStream_t s) {
  GemmParams p = base_params();
  p.A = ws.dZT; p.lda = ws.KT;
  p.B = ws.HcT; p.ldb = ws.KT;
  p.M = V; p.N = d; p.dyn_k = 1; p.meta = ws.unit();
  p.group_m = kGroupMdW;
  p.out = dW; p.ldo = V;
  k_gemm4w<EPI_F32_ACCUM, BGPO_TILE4><<<grid, kGemmThreads4, 0, s>>>(p);
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

// ---- test hook: the GEMM core alone, C[m][n] = sum_k A[m][k] B[n][k] in fp32 ----
extern "C" int bgpo_test_gemm_nt(const uint16_t* A, const uint16_t* B, float* C, int32_t M, int32_t N,
                                 int32_t K, void* stream) {
  using namespace bgpo;
  if (!A || !B || !C || M <= 0 || N <= 0 || K <= 0 || K % 64) return -1;
  // the production kernel stores C^T of its operands' product: swap them
  GemmParams p = base_params();
  p.A = B; p.lda = K; p.B = A; p.ldb = K;
  p.M = N; p.N = M; p.K = K; p.k_split = K;
  p.out = C; p.ldo = N;
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return -3;
  k_gemm4w<EPI_F32_STORE, BGPO_TILE4><<<gemm_grid(dev), kGemmThreads4, 0, (hipStream_t)stream>>>(p);
  return hipGetLastError() == hipSuccess ? 0 : -3;
}

// ---- test hook: tile-configuration variants of the GEMM core (fp32 store) ----
extern "C" int bgpo_test_gemm_variant(const uint16_t* A, const uint16_t* B, float* C, int32_t M,
                                      int32_t N, int32_t K, int32_t variant, int32_t flags,
                                      void* stream) {
  using namespace bgpo;
  if (!A || !B || !C || M <= 0 || N <= 0 || K <= 0 || K % 64) return -1;
  GemmParams p = base_params();
  p.A = A; p.lda = K; p.B = B; p.ldb = K;
  p.M = M; p.N = N; p.K = K; p.k_split = K;
  p.out = C; p.ldo = N;
  p.group_m = (flags & 1) ? M : 1;
  p.plain_order = (flags >> 1) & 1;
  if ((flags >> 8) & 0xFF) p.group_m = (flags >> 8) & 0xFF;
  const int nsplit = (flags >> 16) & 0xFF;
  if (nsplit > 1) {
    p.n_split = nsplit;
    p.k_split = ((K + nsplit - 1) / nsplit + 63) / 64 * 64;
    p.split_stride = (int64_t)M * N;   // C must hold nsplit x M x N floats
  }
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return -3;
  const int cus = gemm_grid(dev);
  hipStream_t s = (hipStream_t)stream;
  switch (variant) {
    case 0: k_gemm<EPI_F32_STORE, 256, 256, 32, 128, 128, 4><<<cus, 256, 0, s>>>(p); break;
    case 1: k_gemm<EPI_F32_STORE, 256, 256, 32, 128, 128, 5><<<cus, 256, 0, s>>>(p); break;
    case 2: k_gemm<EPI_F32_STORE, 256, 256, 64, 128, 128, 2><<<cus, 256, 0, s>>>(p); break;
    case 3: k_gemm<EPI_F32_STORE, 256, 128, 32, 128, 64, 3, 2><<<2 * cus, 256, 0, s>>>(p); break;
    case 4: k_gemm<EPI_F32_STORE, 128, 256, 32, 64, 128, 3, 2><<<2 * cus, 256, 0, s>>>(p); break;
    case 5: k_gemm<EPI_F32_STORE, 256, 256, 64, 128, 64, 2><<<cus, 512, 0, s>>>(p); break;
    case 6: k_gemm<EPI_F32_STORE, 256, 256, 64, 64, 128, 2><<<cus, 512, 0, s>>>(p); break;
    case 7: k_gemm<EPI_F32_STORE, 256, 256, 64, 128, 128, 2, 1, 1><<<cus, 256, 0, s>>>(p); break;
    case 8: k_gemm<EPI_F32_STORE, 256, 256, 64, 128, 64, 2, 1, 1><<<cus, 512, 0, s>>>(p); break;
    case 9: k_gemm<EPI_F32_STORE, 256, 256, 32, 128, 64, 4><<<cus, 512, 0, s>>>(p); break;
    case 10: k_gemm<EPI_F32_STORE, 256, 256, 32, 128, 64, 5><<<cus, 512, 0, s>>>(p); break;
    case 11: k_gemm<EPI_F32_STORE, 256, 256, 64, 64, 128, 2, 1, 1><<<cus, 512, 0, s>>>(p); break;
    case 12: k_gemm<EPI_F32_STORE, 256, 128, 32, 128, 64, 3, 2, 1><<<2 * cus, 256, 0, s>>>(p); break;
    case 13: k_gemm<EPI_F32_STORE, 128, 256, 32, 64, 128, 3, 2, 1><<<2 * cus, 256, 0, s>>>(p); break;
    case 14: k_gemm<EPI_F32_STORE, 256, 256, 32, 128, 128, 4, 1, 1><<<cus, 256, 0, s>>>(p); break;
    case 15: k_gemm<EPI_F32_STORE, 256, 256, 32, 128, 128, 5, 1, 1><<<cus, 256, 0, s>>>(p); break;
    case 16: k_gemm<EPI_F32_STORE, 256, 256, 32, 128, 64, 4, 1, 1><<<cus, 512, 0, s>>>(p); break;
    case 17: k_gemm<EPI_F32_STORE, 256, 256, 32, 128, 64, 5, 1, 1><<<cus, 512, 0, s>>>(p); break;
    case 18:     // the production kernel: it stores C^T of its operands' product
    case 19: {   // the same on a four-stage ring of 32-deep slabs
      GemmParams q = p;
      q.A = B; q.B = A; q.M = N; q.N = M;
      if (!(flags & 1) && !((flags >> 8) & 0xFF)) q.group_m = 1;
      else if (flags & 1) q.group_m = N;
      if (variant == 18)
        k_gemm4w<EPI_F32_STORE, BGPO_TILE4><<<cus, kGemmThreads4, 0, s>>>(q);
      else
        k_gemm4w<EPI_F32_STORE, 256, 256, 32, 4, 1><<<cus, kGemmThreads4, 0, s>>>(q);
      break;
    }
    default: return -1;
  }
  return hipGetLastError() == hipSuccess ? 0 : -3;
}
