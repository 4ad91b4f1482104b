// Grouped bf16 GEMM, second design: direct global->LDS loads (16 bytes per lane,
// no staging registers) into a ring of STAGES LDS buffers, XOR-swizzled tile
// layouts, and MFMA operand fragments read with ds_read_b128 (K-contiguous
// tiles) or with the transposing ds_read_b64_tr_b16 (N-contiguous tiles).
//
// Same problem statement and tile schedule as grouped_gemm in gemm.hpp:
//   C[m][n] = sum_k A[m][k] B[n][k] per expert; GROUP_M groups rows (tokens),
//   GROUP_K groups the contraction (tokens) for weight gradients.
// Operand storage:
//   A_T = false: A[m][k] at A[m*lda + k]        A_T = true: A[m][k] at A[k*lda + m]
//   B_T = false: B[n][k] at B[n*ldb + k]        B_T = true: B[n][k] at B[k*ldb + n]
//
// LDS tile layouts (bf16, 16-byte chunks; BK = 32 or 64):
//   K-contiguous tile [R][BK]: row r holds BK/8 chunks; chunk c of row r is stored
//     at position c ^ swz(r).  A wave's load instruction fills 1024/(2 BK) whole rows.
//   N-contiguous tile [BK][R]: row k holds R/8 chunks; chunk c of row k is stored
//     at position c ^ (4 * (k % 4)) (R >= 128).  An instruction fills 1024/(2R) rows.
// Rows beyond the valid m/n range are loaded from a clamped address (their output
// is never stored); k rows beyond the valid range (GROUP_K tail) are zeroed in LDS.
#pragma once

#include "gemm.hpp"

namespace dmoe {

typedef __attribute__((address_space(3))) void* lds_ptr_t;
typedef short s16x4_t __attribute__((ext_vector_type(4)));

// Direct global->LDS load of 16 bytes per lane into the wave's 1 KiB at lds_wave_base,
// from a wave-uniform base and a 32-bit per-lane byte offset (the scalar-base form: one
// address register per load).  Written out as the instruction (M0 = the wave's LDS
// destination, one wait state before the load reads it) rather than through the
// compiler builtin, so the compiler does not track it and adds no waits of its own:
//   * it cannot tell the LDS operand of a transposing read (ds_read_b64_tr_b16) apart
//     from these loads' destinations and would drain every outstanding load
//     (vmcnt(0)) before each such read, serialising the ring;
//   * its waits for the epilogue's own loads (bias, h, old parameters) then count only
//     those loads; in-order retirement makes them cover the ring loads issued before.
// The pipeline's counted vmcnt waits and barriers order these loads.
// The LDS destination is lds_base + LOFF, LOFF a compile-time byte offset, so one
// scalar register serves every load of a stage.  The scalar add writes SCC, declared
// clobbered: the compiler may otherwise hold a compare result, or the carry of a 64-bit
// address add split around the statement, in SCC across it.
template <int LOFF>
__device__ __forceinline__ void g2l_16_at(const bf16* base, uint32_t off_bytes, char* lds_base) {
  const uint32_t m = (uint32_t)(uintptr_t)(lds_ptr_t)lds_base;
  asm volatile("s_add_u32 m0, %2, %3\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1"
               :: "v"(off_bytes), "s"(base), "s"(m), "i"(LOFF) : "memory", "m0", "scc");
}

// f(integral_constant<int, 0>) ... f(integral_constant<int, N-1>), in order
template <int N, int I = 0, typename F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (I < N) {
    f(std::integral_constant<int, I>{});
    static_for<N, I + 1>(f);
  }
}

// s_waitcnt vmcnt(n) with expcnt/lgkmcnt left free (gfx9 encoding).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

// Workgroup barrier without a memory fence: orders this wave's LDS accesses
// (lgkmcnt) but leaves global loads in flight; LDS data written by the direct
// loads is covered by the explicit vmcnt waits before it.
__device__ __forceinline__ void block_sync_lds() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// Chunk swizzle of a K-contiguous tile.  BK = 64 (8 chunks, 128-byte rows):
// position = chunk ^ (r % 8) or ^ ((r / 2) % 8).  BK = 32 (4 chunks, 64-byte rows):
// position = chunk ^ ((r / 4) % 4), which makes any 16 consecutive rows read at one
// chunk fall on 16 distinct 16-byte bank groups.
template <int BK, int SW>
__device__ __forceinline__ int swz_kc(int r) {
  if constexpr (BK == 32) return (r >> 2) & 3;
  return SW == 0 ? (r & 7) : ((r >> 1) & 7);
}

// ---- K-contiguous tile [R][BK] -------------------------------------------------------
template <int R, int NW, int SW, int BK>
struct KcTile {
  static constexpr int RB = BK * 2;                    // bytes per row
  static constexpr int CH = BK / 8;                    // chunks per row
  static constexpr int RPI = 1024 / RB;                // rows per wave instruction
  static constexpr int BYTES = R * RB;
  static constexpr int INSTR = R / RPI;                // 1 KB wave instructions per tile
  static constexpr int PER_WAVE = (INSTR + NW - 1) / NW;
  static_assert(BK == 32 || BK == 64, "BK");
  static_assert(R % RPI == 0, "rows");
  // issue this wave's loads: rows [0, R) of the tile starting at `base` (row stride ld)
  __device__ __forceinline__ static void load(const bf16* base, int64_t ld, int rvalid, char* lds, int wave,
                                              int lane) {
    char* lw = lds + wave * 1024;
    static_for<PER_WAVE>([&](auto I) {
      constexpr int i = decltype(I)::value;
      const int q = wave + i * NW;
      if (INSTR % NW != 0 && q >= INSTR) return;
      const int r = q * RPI + lane / CH;
      const int c = (lane % CH) ^ swz_kc<BK, SW>(r);
      const int rr = r < rvalid ? r : rvalid - 1;
      g2l_16_at<i * NW * 1024>(base, ((uint32_t)rr * (uint32_t)ld + (uint32_t)(c * 8)) * 2u, lw);
    });
  }
  // fragment of rows r0 + (lane % 32), k chunk kc + lane / 32 (8 bf16)
  __device__ __forceinline__ static bf16x8_t frag(const char* lds, int r0, int kc, int lane) {
    const int r = r0 + (lane & 31);
    const int c = (kc + (lane >> 5)) ^ swz_kc<BK, SW>(r);
    return *reinterpret_cast<const bf16x8_t*>(lds + r * RB + c * 16);
  }
  // The same fragment split into a per-lane part and a per-fragment constant: the
  // swizzle repeats every 16 rows, so for r0 a multiple of 16 the byte offset is
  // r0 * RB + lane_off(kc, lane), the second term the same for every r0.
  __device__ __forceinline__ static uint32_t lane_off(int kc, int lane) {
    const int r = lane & 31;
    return (uint32_t)(r * RB + (((kc + (lane >> 5)) ^ swz_kc<BK, SW>(r)) << 4));
  }
  __device__ __forceinline__ static bf16x8_t frag_at(const char* lds, int r0, uint32_t off) {
    return *reinterpret_cast<const bf16x8_t*>(lds + r0 * RB + off);
  }
};

// ---- N-contiguous tile [BK][R] (row = k) ---------------------------------------------
template <int R, int NW, int BK>
struct NcTile {
  static constexpr int BYTES = BK * R * 2;
  static constexpr int CPR = R / 8;                    // chunks per row
  static constexpr int RPI = 1024 / (R * 2);           // rows per wave instruction
  static constexpr int INSTR = BK / RPI;
  static constexpr int PER_WAVE = (INSTR + NW - 1) / NW;
  static_assert(R >= 128 && R <= 512 && (R & (R - 1)) == 0, "cols");
  __device__ __forceinline__ static int swz(int k) { return 4 * (k & 3); }
  // element (col c, k) at base[k * ld + c]; rows k >= kvalid clamped (zeroed later)
  __device__ __forceinline__ static void load(const bf16* base, int64_t ld, int cvalid, int kvalid, char* lds,
                                              int wave, int lane) {
    char* lw = lds + wave * 1024;
    static_for<PER_WAVE>([&](auto I) {
      constexpr int i = decltype(I)::value;
      const int q = wave + i * NW;
      if (INSTR % NW != 0 && q >= INSTR) return;
      const int k = q * RPI + lane / CPR;
      const int pos = lane % CPR;
      const int c = pos ^ swz(k);
      int col = c * 8;
      col = col < cvalid ? col : ((cvalid - 1) & ~7);
      const int kk = k < kvalid ? k : kvalid - 1;
      g2l_16_at<i * NW * 1024>(base, ((uint32_t)kk * (uint32_t)ld + (uint32_t)col) * 2u, lw);
    });
  }
  // zero rows [kvalid, kend) of the tile (GROUP_K tail)
  __device__ __forceinline__ static void zero_tail(char* lds, int kvalid, int kend, int tid, int nt) {
    uint4* p = reinterpret_cast<uint4*>(lds + kvalid * R * 2);
    const int n = (kend - kvalid) * CPR;
    for (int i = tid; i < n; i += nt) p[i] = make_uint4(0, 0, 0, 0);
  }
  // MFMA fragment for columns c0 .. c0+31 (lane % 32) and k = kk .. kk+15 (lane / 32 picks 8):
  // two transposing reads, 4 k each.
  __device__ __forceinline__ static bf16x8_t frag(const char* lds, int c0, int kk, int lane) {
    const int g = lane >> 4, i = lane & 15;
    const int col = c0 + 16 * (g & 1) + 4 * (i & 3);
    const int chunk = col >> 3, within = (col & 7) * 2;
    s16x4_t lo, hi;
    {
      const int k = kk + 8 * (g >> 1) + (i >> 2);
      const char* a = lds + k * (R * 2) + ((chunk ^ swz(k)) << 4) + within;
      lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4_t*)(a));
    }
    {
      const int k = kk + 8 * (g >> 1) + 4 + (i >> 2);
      const char* a = lds + k * (R * 2) + ((chunk ^ swz(k)) << 4) + within;
      hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s16x4_t*)(a));
    }
    typedef short s16x8_t __attribute__((ext_vector_type(8)));
    s16x8_t v = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
    return __builtin_bit_cast(bf16x8_t, v);
  }
  // The same fragment for columns 32 m .. 32 m + 31 split into a per-lane part and a
  // k-dependent constant: kk a multiple of 16 leaves the swizzle 4 (k % 4) unchanged,
  // so the lower read is at kk * 2R + lane_off(m, lane) and the upper one 4 rows on.
  __device__ __forceinline__ static uint32_t lane_off(int m, int lane) {
    const int g = lane >> 4, i = lane & 15;
    const int col = 32 * m + 16 * (g & 1) + 4 * (i & 3);
    const int k = 8 * (g >> 1) + (i >> 2);
    return (uint32_t)(k * (R * 2) + (((col >> 3) ^ swz(k)) << 4) + (col & 7) * 2);
  }
  __device__ __forceinline__ static bf16x8_t frag_at(const char* lds, int kk, uint32_t off) {
    const s16x4_t lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (__attribute__((address_space(3))) s16x4_t*)(lds + kk * (R * 2) + off));
    const s16x4_t hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (__attribute__((address_space(3))) s16x4_t*)(lds + (kk + 4) * (R * 2) + off));
    typedef short s16x8_t __attribute__((ext_vector_type(8)));
    s16x8_t v = {lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
    return __builtin_bit_cast(bf16x8_t, v);
  }
};

// The tile plan and the expert offsets are written by earlier kernels and only read
// while a GEMM runs.  Read through the constant address space with wave-uniform
// indices they become scalar loads, counted by lgkmcnt: they neither join the vector
// memory queue whose in-order counts the pipeline waits on nor force it to drain.
__device__ __forceinline__ int ld_plan(const int32_t* p, int i) {
  return ((const __attribute__((address_space(4))) int32_t*)p)[i];
}
// expert owning global tile L (tiles of expert e start at tprefix[e] * scale), for a
// tile not below the one whose expert was `hint`
__device__ __forceinline__ int find_group_plan(const int32_t* tprefix, int scale, int groups, int L, int hint) {
  if (ld_plan(tprefix, hint + 1) * scale > L) return hint;
  int lo = hint + 1, hi = groups;   // tprefix[lo]*scale <= L < tprefix[hi]*scale
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (ld_plan(tprefix, mid) * scale <= L) lo = mid; else hi = mid;
  }
  return lo;
}

// Runtime-selected s_waitcnt vmcnt(n) for n in [0, 63] (n is wave-uniform).
__device__ __forceinline__ void wait_vmcnt_rt(int n) {
  if (n >= 48) { if (n >= 56) wait_vmcnt<56>(); else wait_vmcnt<48>(); }
  else if (n >= 32) { if (n >= 40) wait_vmcnt<40>(); else wait_vmcnt<32>(); }
  else if (n >= 16) { if (n >= 24) wait_vmcnt<24>(); else wait_vmcnt<16>(); }
  else if (n >= 12) wait_vmcnt<12>();
  else if (n >= 8) wait_vmcnt<8>();
  else if (n >= 4) wait_vmcnt<4>();
  else wait_vmcnt<0>();
}

// How the epilogue writes a bf16 output tile.
//   STORE_DIRECT: each lane stores 16 contiguous bytes of its row straight from its
//     registers (after a lane swap), so one wave instruction writes 32 rows x 32 bytes:
//     every 128-byte line of the output is completed by four instructions.
//   STORE_STAGED: each wave passes 32 rows x 64 columns of its output at a time through
//     4 KiB of LDS of its own and stores whole lines: one wave instruction writes
//     8 rows x 128 bytes.
//   STORE_STAGED_NT: as STORE_STAGED, with the non-temporal hint on the stores.
enum StoreMode { STORE_DIRECT = 0, STORE_STAGED = 1, STORE_STAGED_NT = 2 };
constexpr int STG_WAVE_BYTES = 4096;

// Staging layout of a wave's 32 x 64 piece: row r (0..31) holds 128 bytes, 16-byte
// chunk c at position c ^ ((r / 2) % 8), so the 32 rows written at one chunk and the
// 8 rows read per instruction spread over the LDS banks.
__device__ __forceinline__ int stg_off(int r, int c) { return r * 128 + ((c ^ ((r >> 1) & 7)) << 4); }

// Schedule of one tile, per wave:
//   * the prologue issues every stage of the LDS ring (the ring is free once the
//     previous tile's reads are done), before the previous tile's epilogue;
//   * stage kt is consumed in BK/16 MFMA steps; the fragments of step kk+1 are read
//     while the MFMAs of step kk run, and in the last step the wave waits for stage
//     kt+1, passes the barrier, refills the ring slot of stage kt with stage
//     kt+STAGES and reads the first fragments of stage kt+1, all before issuing the
//     last MFMAs of stage kt, so no LDS latency is exposed at stage boundaries (the
//     row-grouped GEMMs with N-contiguous weights issue those MFMAs before the wait
//     instead, see MM_EARLY);
//   * vector-memory operations (loads, stores, direct-to-LDS loads) retire from the
//     vmcnt counter in issue order on gfx9-family chips, so "stage s has landed" is
//     vmcnt <= (operations issued after stage s).  The previous tile's epilogue stores
//     follow the prologue stages; they are counted only when that tile was full
//     (exact count known), otherwise the wait also covers them.
// Rows of a tile are split in 32-row blocks; block b belongs to wave row wm = b % WM
// as its block j = b / WM, so a partly filled tile (the last m-tile of an expert)
// spreads its live blocks over all wave rows and SIMDs.  Each wave runs a loop
// specialised for its number of live blocks, so the loop body has no branches.
//
// Extra block (XB = 1, GROUP_M with 256 x 256 tiles of 8 waves): a tile holds up to
// 288 rows, the 32 beyond the first 256 forming a ninth row block that all 8 waves
// share, wave (wm, wn) computing its 32 x 32 piece at the wave's own column block wm.
// The wave holds that block's B fragment already (its column block wm), so the piece
// costs one more A fragment read per step; the loop is compiled once per wm, which
// names the fragment at compile time.
// An expert's rows are then split into ceil(rows / 288) tiles of equal block counts, so
// an expert with a few rows more than a multiple of 256 gets no nearly empty tile
// (which would stream the expert's whole weight slab again for those rows).
template <int GM, bool A_T, bool B_T, int EPI, int BM, int BN, int WM, int WN, int STAGES, int SW, int BK,
          int STO = STORE_DIRECT, int XB = 0>
__global__ void __launch_bounds__(64 * WM * WN)
grouped_gemm2(GemmArgs<bf16> p) {
  constexpr int NW = WM * WN, NT = 64 * NW;
  constexpr int WTM = BM / WM, WTN = BN / WN;
  constexpr int TM = WTM / 32, TN = WTN / 32;
  constexpr int KK = BK / 16;
  using TA = typename std::conditional<A_T, NcTile<BM, NW, BK>, KcTile<BM, NW, SW, BK>>::type;
  using TB = typename std::conditional<B_T, NcTile<BN, NW, BK>, KcTile<BN, NW, SW, BK>>::type;
  constexpr int XROWS = XB ? 32 : 0;                 // rows of the extra block
  constexpr int BMT = BM + XROWS;                    // rows a tile can hold
  constexpr int ABYTES = TA::BYTES + XROWS * BK * 2, SBYTES = ABYTES + TB::BYTES;
  constexpr int LPS = TA::PER_WAVE + TB::PER_WAVE;   // load instructions per stage per wave
  // (with XB, waves 0..3 load one more: the extra block's 32 rows, 8 rows each)
  // store instructions of a full tile's epilogue, per wave
  constexpr int SFULL = EPI == EPI_F32 ? TM * TN * 4 : TM * TN * 2 * (EPI == EPI_BIAS_ACT ? 2 : 1);
  static_assert(TM >= 1 && TM <= 5 && TN >= 1, "tile");
  // GROUP_M tiles taller than 256 rows split each expert's rows evenly (in 32-row
  // blocks) over its m-tiles, so an expert slightly above a multiple of the tile height
  // gets no nearly empty last tile
  constexpr bool BAL = GM == GROUP_M && (BM > 256 || XB);
  static_assert(!XB || (GM == GROUP_M && !A_T && BM == 256 && BN == 256 && WM == 4 && WN == 2 && STAGES == 2 &&
                        STO == STORE_DIRECT && EPI != EPI_F32 && EPI != EPI_SGD),
                "extra block: GROUP_M 256 x 256 tiles of 8 waves, 2 stages, direct stores");
  static_assert(KK % 2 == 0, "fragment slots alternate over an even number of steps");
  static_assert(TA::INSTR % NW == 0 && TB::INSTR % NW == 0, "equal load counts per wave");
  static_assert(GM == GROUP_M || (A_T && B_T), "GROUP_K takes both operands stored per token");
  static_assert(STAGES * LPS <= 63, "vmcnt range");
  static_assert(STO == STORE_DIRECT || (EPI != EPI_F32 && WTN % 64 == 0), "staged stores: bf16 output, 64-col pieces");

  extern __shared__ __align__(1024) char smem[];
  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / WN, wn = wave % WN;
  const int lps = LPS + (XB && wave < 4 ? 1 : 0);     // this wave's loads per stage
  // per-lane byte offsets of the MFMA fragments within a stage: K-contiguous tiles by
  // k-step (shared by A and B, whose rows have the same width and swizzle), N-contiguous
  // tiles by 32-column block
  uint32_t kc_off[KK], a_nc[TM], b_nc[TN];
#pragma unroll
  for (int kk = 0; kk < KK; ++kk) kc_off[kk] = KcTile<BM, NW, SW, BK>::lane_off(kk * 2, lane);
  if constexpr (A_T) {
#pragma unroll
    for (int j = 0; j < TM; ++j) a_nc[j] = TA::lane_off(j * WM + wm, lane);
  }
  if constexpr (B_T) {
#pragma unroll
    for (int i = 0; i < TN; ++i) b_nc[i] = TB::lane_off(wn * TN + i, lane);
  }

  const int total = ld_plan(p.tprefix, p.groups) * p.tscale;
  int L, Lend, Lstep;
  if (p.chunked) {
    const int x = blockIdx.x & 7, lb = blockIdx.x >> 3;
    L = (int)(((int64_t)x * total) >> 3) + lb;
    Lend = (int)(((int64_t)(x + 1) * total) >> 3);
    Lstep = (gridDim.x - x + 7) >> 3;
  } else {
    L = blockIdx.x; Lend = total; Lstep = gridDim.x;
  }
  const int NTILES = (p.N + BN - 1) / BN;

  // Coordinates and operand bases of tile L.
  struct TileC {
    int e, off, m0, n0, mvalid, nvalid, kvalid, nk;
    int base;                      // ring slot of the tile's stage 0 (EARLY only; else 0)
    const bf16* Ab;
    const bf16* Bb;
  };
  // Weight-gradient GEMMs with a deep ring: when a tile has fewer k-steps than the ring
  // has slots (few rows per expert), the next tile's first stages are loaded into the
  // free slots before this tile's MFMAs, so their latency hides behind this tile's
  // work and stores instead of being waited for right after them.  Stage s of a tile
  // sits in slot (base + s) % STAGES, base following the previous tile's last stage.
  constexpr bool EARLY = GM == GROUP_K && STAGES > 2;
  auto slot = [&](const TileC& t, int s) -> char* {
    if constexpr (EARLY) return smem + ((t.base + s) % STAGES) * SBYTES;
    else return smem + (s % STAGES) * SBYTES;
  };
  int ehint = 0;                   // group of the previous tile of this block
  auto setup = [&](int Lt) {
    TileC t;
    t.base = 0;
    t.e = find_group_plan(p.tprefix, p.tscale, p.groups, Lt, ehint);
    ehint = t.e;
    const int q = Lt - ld_plan(p.tprefix, t.e) * p.tscale;
    t.off = ld_plan(p.offsets, t.e);
    const int cnt = ld_plan(p.offsets, t.e + 1) - t.off;
    if constexpr (GM == GROUP_M) {
      const int mt_e = (cnt + BMT - 1) / BMT;
      if constexpr (BAL) {
        // m-tile qm holds 32-row blocks [qm B / mt_e, (qm + 1) B / mt_e) of the expert's
        // B blocks: tile sizes differ by at most one block.  Odd experts number their
        // m-tiles backwards, so the persistent blocks that take the same m position
        // expert after expert (tiles are dealt out in a fixed stride) alternate between
        // the larger and the smaller tiles instead of one group falling steadily behind
        // the other, which would stop them sharing each weight slab in L2.
        const int qm = (t.e & 1) ? mt_e - 1 - q % mt_e : q % mt_e;
        if constexpr (B_T) {
          // N-contiguous weights: the expert's rows split evenly, so its m-tiles issue the
          // same number of row blocks and stay in step through the whole k loop, sharing
          // each stage of the weight slab in L2 (a few more rows of padding, measured
          // faster than splitting whole blocks, which is faster for K-contiguous weights)
          const int r0 = qm * cnt / mt_e, r1 = (qm + 1) * cnt / mt_e;
          t.m0 = r0;
          t.mvalid = r1 - r0;
        } else {
          const int nb = (cnt + 31) / 32;
          const int b0 = qm * nb / mt_e, b1 = (qm + 1) * nb / mt_e;
          t.m0 = b0 * 32;
          t.mvalid = cnt - t.m0 < (b1 - b0) * 32 ? cnt - t.m0 : (b1 - b0) * 32;
        }
      } else {
        t.m0 = (q % mt_e) * BM;
        t.mvalid = cnt - t.m0;
      }
      t.n0 = (q / mt_e) * BN;
      t.kvalid = p.K;
      t.Ab = p.A + (int64_t)(t.off + t.m0) * p.lda;
      t.Bb = p.B + (int64_t)t.e * p.b_gstride + (B_T ? (int64_t)t.n0 : (int64_t)t.n0 * p.ldb);
    } else {
      // grouped order: consecutive tiles walk GMT m-tiles, then the next n-tile, so the
      // tiles in flight on one XCD share a few A and B slabs (fits its L2)
      constexpr int GMT = 4;
      const int MTILES = (p.M + BM - 1) / BM;
      const int per_group = GMT * NTILES;
      const int first = (q / per_group) * GMT;
      const int gsize = MTILES - first < GMT ? MTILES - first : GMT;
      const int qi = q % per_group;
      t.m0 = (first + qi % gsize) * BM; t.n0 = (qi / gsize) * BN;
      t.mvalid = p.M - t.m0; t.kvalid = cnt;
      t.Ab = p.A + (int64_t)t.off * p.lda + t.m0;
      t.Bb = p.B + (int64_t)t.off * p.ldb + t.n0;
    }
    t.nvalid = p.N - t.n0;
    t.nk = (t.kvalid + BK - 1) / BK;
    return t;
  };
  auto issue = [&](const TileC& t, int kt) {
    char* buf = slot(t, kt);
    const int k0 = kt * BK;
    if constexpr (A_T) TA::load(t.Ab + (int64_t)k0 * p.lda, p.lda, t.mvalid, t.kvalid - k0, buf, wave, lane);
    else TA::load(t.Ab + k0, p.lda, t.mvalid, buf, wave, lane);
    if constexpr (XB) {
      // rows BM .. BM+31 of the tile: wave w < 4 loads rows BM + 8w .. BM + 8w + 7
      if (wave < 4) {
        constexpr int CH = BK / 8;
        const int r = BM + wave * (1024 / (BK * 2)) + lane / CH;
        const int c = (lane % CH) ^ swz_kc<BK, SW>(r);
        const int rr = r < t.mvalid ? r : t.mvalid - 1;
        g2l_16_at<0>(t.Ab + k0, ((uint32_t)rr * (uint32_t)p.lda + (uint32_t)(c * 8)) * 2u,
                     buf + TA::BYTES + wave * 1024);
      }
    }
    if constexpr (B_T) TB::load(t.Bb + (int64_t)k0 * p.ldb, p.ldb, t.nvalid, t.kvalid - k0, buf + ABYTES, wave, lane);
    else TB::load(t.Bb + k0, p.ldb, t.nvalid, buf + ABYTES, wave, lane);
  };
  auto prologue = [&](const TileC& t) {
#pragma unroll
    for (int s = 0; s < STAGES; ++s)
      if (s < t.nk) issue(t, s);
  };
  // stage s of tile t has landed in this wave's view; `after` = load stages issued after it
  auto wait_stage = [&](int after, int extra) { wait_vmcnt_rt(after * lps + extra > 63 ? 63 : after * lps + extra); };
  // GROUP_K: zero the k rows of stage s past the expert's tokens, once every wave's loads
  // landed, up to the end of the last 16-deep MFMA step that reads any row of the
  // expert (the steps past it are not issued)
  auto fix_tail = [&](const TileC& t, int s) {
    if constexpr (GM == GROUP_K) {
      const int kv = t.kvalid - s * BK;
      if (kv < BK) {
        const int kend = (kv + 15) / 16 * 16;
        char* buf = slot(t, s);
        block_sync_lds();
        if (kend > kv) {
          TA::zero_tail(buf, kv, kend, tid, NT);
          TB::zero_tail(buf + ABYTES, kv, kend, tid, NT);
        }
      }
    }
  };

  TileC nxt{};
  if (L < Lend) {
    nxt = setup(L);
    prologue(nxt);
  }
  int prev_stores = 0;            // exact store count of the previous epilogue, 0 if unknown
  for (; L < Lend; L += Lstep) {
    const TileC t = nxt;
    const int e = t.e, off = t.off, m0 = t.m0, n0 = t.n0, mvalid = t.mvalid, nvalid = t.nvalid;
    const int nk = t.nk;
    const bool more = L + Lstep < Lend;
    int early = 0;                 // stages of the next tile issued before this tile's MFMAs
    const int nblk_all = (mvalid + 31) / 32;             // live 32-row blocks of the tile
    const int nblk = nblk_all < BM / 32 ? nblk_all : BM / 32;
    const bool xl = XB && nblk_all > BM / 32;            // the extra block is live
    int nl = (nblk - wm + WM - 1) / WM;                  // of them, this wave's (a prefix of j)
    nl = nl < 0 ? 0 : (nl > TM ? TM : nl);

    f32x16_t acc[TN][TM];
#pragma unroll
    for (int i = 0; i < TN; ++i)
#pragma unroll
      for (int j = 0; j < TM; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;
    f32x16_t accx;                                       // the extra block's piece
#pragma unroll
    for (int r = 0; r < 16; ++r) accx[r] = 0.f;

    auto mainloop = [&](auto NLc, auto XLc, auto XCc) {
      constexpr int NL = decltype(NLc)::value;
      constexpr bool XL = decltype(XLc)::value;
      constexpr int XC = decltype(XCc)::value;
      static_assert(!XL || XC < TN, "extra block column within the wave's columns");
      constexpr int NDS = (A_T ? 2 : 1) * NL + (B_T ? 2 : 1) * TN + (XL ? 1 : 0);
      bf16x8_t fa[2][TM], fb[2][TN], fax[2];
      auto ldfrag = [&](const char* buf, int kk, int slot) {
        if constexpr (NL == 0) return;             // no rows: nothing to multiply
        const char* as = buf;
        const char* bs = buf + ABYTES;
        if constexpr (XL) fax[slot] = TA::frag_at(as, BM, kc_off[kk]);
#pragma unroll
        for (int j = 0; j < NL; ++j) {
          const int r0 = (j * WM + wm) * 32;
          if constexpr (A_T) fa[slot][j] = TA::frag_at(as, kk * 16, a_nc[j]);
          else fa[slot][j] = TA::frag_at(as, r0, kc_off[kk]);
        }
#pragma unroll
        for (int i = 0; i < TN; ++i) {
          if constexpr (B_T) fb[slot][i] = TB::frag_at(bs, kk * 16, b_nc[i]);
          else fb[slot][i] = TB::frag_at(bs, wn * WTN + i * 32, kc_off[kk]);
        }
      };
      auto mm = [&](int slot) {
#pragma unroll
        for (int j = 0; j < NL; ++j)
#pragma unroll
          for (int i = 0; i < TN; ++i)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fb[slot][i], fa[slot][j], acc[i][j], 0, 0, 0);
        // the extra block's columns are the wave's column block wm (XC, its
        // compile-time copy): its B fragment is fb[slot][XC]
        if constexpr (XL) accx = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fb[slot][XC], fax[slot], accx, 0, 0, 0);
      };
      auto interleave = [&]() {
#pragma unroll
        for (int q = 0; q < NL * TN + (XL ? 1 : 0); ++q) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);                 // one MFMA
          if (q < NDS) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);   // one LDS read
        }
      };
      // stage 0: issued in the prologue, followed by the load stages 1.. and the
      // previous tile's epilogue stores
      {
        const int issued = nk < STAGES ? nk : STAGES;
        wait_stage(issued - 1, prev_stores);
        fix_tail(t, 0);
        block_sync_lds();
        ldfrag(slot(t, 0), 0, 0);
      }
      if constexpr (EARLY) {
        // every stage of this tile is already issued and the slots past its last one
        // held the previous tile's stages, consumed before the previous tile's final
        // barrier: fill them with the next tile's first stages
        if (more && nk < STAGES) {
          nxt = setup(L + Lstep);
          nxt.base = (t.base + nk) % STAGES;
          early = nxt.nk < STAGES - nk ? nxt.nk : STAGES - nk;
          for (int st = 0; st < early; ++st) issue(nxt, st);
        }
      }
      // every stage but the last: the last MFMA step also moves on to the next stage
      for (int kt = 0; kt + 1 < nk; ++kt) {
        const char* cur = slot(t, kt);
#pragma unroll
        for (int kk = 0; kk + 1 < KK; ++kk) {
          ldfrag(cur, kk + 1, (kk & 1) ^ 1);
          mm(kk & 1);
          interleave();
        }
        // Row-grouped GEMMs with N-contiguous weights (transposing fragment reads) issue
        // the stage's last MFMA step before the wait for the next stage, keeping the MFMA
        // pipe busy while the loads land; the first fragments of the next stage are then
        // read after the barrier with nothing to hide their latency behind.  Measured
        // 3-4% faster for those GEMMs and 2% slower for the others, which keep the last
        // step after the barrier to cover those fragment reads.
        constexpr bool MM_EARLY = STAGES == 2 && GM == GROUP_M && B_T;
        if constexpr (MM_EARLY) mm(1);
        if constexpr (STAGES == 2) {
          // stage kt+1 is the newest load stage; only at kt = 0 do the previous
          // epilogue's stores follow it (a compile-time wait in the steady state)
          if (kt == 0) wait_vmcnt_rt(prev_stores);
          else wait_vmcnt<0>();
        } else {
          // stages issued after kt+1: up to kt+STAGES-1, capped by the last stage; the
          // previous epilogue's stores come after the prologue stages 0..STAGES-1
          const int last = kt + STAGES - 1 < nk - 1 ? kt + STAGES - 1 : nk - 1;
          // (the next tile's early stages were issued after all of this tile's)
          wait_stage(last - (kt + 1), (kt + 1 < STAGES ? prev_stores : 0) + early * LPS);
        }
        fix_tail(t, kt + 1);
        block_sync_lds();               // every wave is done with slot kt and sees stage kt+1
        if (kt + STAGES < nk) issue(t, kt + STAGES);
        ldfrag(slot(t, kt + 1), 0, 0);
        if constexpr (!MM_EARLY) {
          mm(1);
          interleave();
        }
      }
      {
        // the last stage; with GROUP_K only its MFMA steps that reach a row of the
        // expert (rows past the last are zero and would add nothing)
        const char* cur = slot(t, nk - 1);
        const int nkk = GM == GROUP_K ? (t.kvalid - (nk - 1) * BK + 15) / 16 : KK;
#pragma unroll
        for (int kk = 0; kk + 1 < KK; ++kk) {
          if (kk + 1 < nkk) ldfrag(cur, kk + 1, (kk & 1) ^ 1);
          if (kk < nkk) mm(kk & 1);
          interleave();
        }
        if (KK - 1 < nkk) mm(1);
      }
    };
    using NoX = std::integral_constant<bool, false>;
    using C0 = std::integral_constant<int, 0>;
    using XLt = std::integral_constant<bool, (XB != 0)>;
    using TMt = std::integral_constant<int, TM>;
    if (XB && xl) {
      static_assert(!XB || WM == 4, "four wave rows");
      if (wm == 0) mainloop(TMt{}, XLt{}, C0{});
      else if (wm == 1) mainloop(TMt{}, XLt{}, std::integral_constant<int, 1>{});
      else if (wm == 2) mainloop(TMt{}, XLt{}, std::integral_constant<int, (XB ? 2 : 0)>{});
      else mainloop(TMt{}, XLt{}, std::integral_constant<int, (XB ? 3 : 0)>{});
    }
    else if (nl == TM) mainloop(TMt{}, NoX{}, C0{});
    else if (TM >= 2 && nl == 1) mainloop(std::integral_constant<int, 1>{}, NoX{}, C0{});
    else if (TM >= 3 && nl == 2) mainloop(std::integral_constant<int, (TM >= 3 ? 2 : 1)>{}, NoX{}, C0{});
    else if (TM >= 4 && nl == 3) mainloop(std::integral_constant<int, (TM >= 4 ? 3 : 1)>{}, NoX{}, C0{});
    else if (TM >= 5 && nl == 4) mainloop(std::integral_constant<int, (TM >= 5 ? 4 : 1)>{}, NoX{}, C0{});
    else mainloop(std::integral_constant<int, 0>{}, NoX{}, C0{});

    block_sync_lds();      // every wave is done with the ring before the next tile's loads

    // Epilogue operands read from memory are loaded before the next tile's loads where
    // registers allow: vector-memory operations retire in issue order, so a load issued
    // after the prologue waits for it.  The bias (one row, TN x 4 values) is loaded
    // first.  The activation derivative reads a whole tile of h, too large to hold
    // next to the accumulators; its loads follow only the first stage of the next tile,
    // and the remaining stages are issued after the epilogue.
    const int l32 = lane & 31, lhi = lane >> 5;
    constexpr bool HAS_BIAS = EPI == EPI_BIAS || EPI == EPI_BIAS_ACT;
    constexpr bool HAS_AUX = EPI == EPI_DACT || EPI == EPI_SGD;   // reads a tile in C's layout
    constexpr int PRE = HAS_AUX ? 1 : STAGES;       // prologue stages issued before the epilogue
    uint2 bias_v[HAS_BIAS ? TN : 1][4];
    if constexpr (HAS_BIAS) {
#pragma unroll
      for (int i = 0; i < TN; ++i)
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int nl_ = wn * WTN + i * 32 + 8 * g + 4 * lhi;
          const int n = n0 + (nl_ < nvalid ? nl_ : 0);
          bias_v[i][g] = *reinterpret_cast<const uint2*>(p.bias + (int64_t)e * p.bias_gstride + n);
        }
    }
    uint2 bias_x[4];                                     // the extra block's columns
    if constexpr (XB && HAS_BIAS) {
      if (xl) {
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int nl_ = wn * WTN + wm * 32 + 8 * g + 4 * lhi;
          bias_x[g] = *reinterpret_cast<const uint2*>(p.bias + (int64_t)e * p.bias_gstride + n0 +
                                                      (nl_ < nvalid ? nl_ : 0));
        }
      }
    }

    // SGD with staged stores on a 2-slot ring: ring slot 1 is idle until the next tile's
    // stage 1 is issued after the epilogue, so each wave passes its fp32 accumulators
    // through 8 KiB of it, 32 rows x 64 columns at a time, and the update is computed in
    // the store layout: lane L handles row L/8 + 8q, columns 8(L%8) .. +7 of the piece,
    // reading the old parameters as whole 128-byte lines one piece ahead of their use.
    constexpr bool SGD_SLOT = EPI == EPI_SGD && STO != STORE_DIRECT && STAGES == 2 && GM == GROUP_K;
    static_assert(!SGD_SLOT || (NW * 8192 <= SBYTES && WTN % 64 == 0), "fp32 staging in one ring slot");
    char* s32 = smem + SBYTES + wave * 8192;
    // element (r, c) of the 32 x 64 fp32 piece: 16-byte chunk c/4 of row r, XOR-swizzled
    auto s32_off = [](int r, int ch) { return r * 256 + ((ch ^ (r & 15)) << 4); };
    constexpr int HP = TN >= 2 ? TN / 2 : 1;    // 64-column pieces per 32-row block
    const int np = nl * HP;                      // this wave's pieces (uniform)
    bf16* W = reinterpret_cast<bf16*>(p.C);
    auto prow = [&](int pc, int qd) {            // parameter row offset of lane's row qd
      const int ml = ((pc / HP) * WM + wm) * 32 + (lane >> 3) + 8 * qd;
      return (int64_t)e * p.c_gstride + (int64_t)(m0 + (ml < mvalid ? ml : 0)) * p.ldc;
    };
    auto pcol = [&](int pc) {
      const int col = wn * WTN + 64 * (pc % HP) + 8 * (lane & 7);
      return n0 + (col < nvalid ? col : 0);
    };
    // the parameter loads are issued for every lane (clamped in range); stores only
    // where the row and column are valid.  With non-temporal stores the old parameters
    // are read with the same hint: each is read once, and like the new values it then
    // streams past the L2 instead of evicting the GEMM's operands.
    uint4 wold[2][4];
    auto load_piece = [&](int pc, uint4 (&dst)[4]) {
      typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
#pragma unroll
      for (int qd = 0; qd < 4; ++qd) {
        const bf16* src = W + prow(pc, qd) + pcol(pc);
        if constexpr (STO == STORE_STAGED_NT)
          dst[qd] = __builtin_bit_cast(uint4, __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(src)));
        else
          dst[qd] = *reinterpret_cast<const uint4*>(src);
      }
    };
    if (more) {
      if (early == 0) {
        nxt = setup(L + Lstep);
        if constexpr (EARLY) nxt.base = (t.base + nk) % STAGES;
      }
#pragma unroll
      for (int st = early; st < PRE; ++st)
        if (st < nxt.nk) issue(nxt, st);
    }

    // epilogue (same accumulator layout as grouped_gemm); stores issued by this wave
    // number SFULL exactly when every row and column of its part of the tile is valid
    constexpr int SXB = 2 * (EPI == EPI_BIAS_ACT ? 2 : 1);   // stores of the extra block's piece
    const bool full = nl == TM && mvalid >= (xl ? BMT : BM) && nvalid >= BN;
    prev_stores = full ? SFULL + (xl ? SXB : 0) : 0;

    // One 32 x 32 block in C's layout, straight from registers: lane (row l32, half lhi)
    // holds columns cb + 8g + 4 lhi .. +3 of row crow for g = 0..3 (bias bv and the tile
    // read in C's layout av per column group).
    auto emit_direct = [&](const f32x16_t& a, int cb, int64_t crow, bool mok, const uint2 (&bv)[4],
                           const uint2 (&av)[4]) {
      uint32_t pk[4][2], pa[4][2];      // bf16 pairs of column group g (output, activation)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int nl_ = cb + 8 * g + 4 * lhi;
        const int n = n0 + nl_;
        float v[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) v[r] = a[4 * g + r];
        if constexpr (HAS_BIAS) {
          const uint2 b = bv[g];
          v[0] += __uint_as_float(b.x << 16); v[1] += __uint_as_float(b.x & 0xffff0000u);
          v[2] += __uint_as_float(b.y << 16); v[3] += __uint_as_float(b.y & 0xffff0000u);
        }
        if constexpr (EPI == EPI_DACT) {
          const uint2 hv = av[g];
          v[0] *= act_bwd_fast(__uint_as_float(hv.x << 16), p.act);
          v[1] *= act_bwd_fast(__uint_as_float(hv.x & 0xffff0000u), p.act);
          v[2] *= act_bwd_fast(__uint_as_float(hv.y << 16), p.act);
          v[3] *= act_bwd_fast(__uint_as_float(hv.y & 0xffff0000u), p.act);
        }
        if constexpr (EPI == EPI_SGD) {
          const uint2 wv = av[g];
          v[0] = __uint_as_float(wv.x << 16) - p.lr * v[0];
          v[1] = __uint_as_float(wv.x & 0xffff0000u) - p.lr * v[1];
          v[2] = __uint_as_float(wv.y << 16) - p.lr * v[2];
          v[3] = __uint_as_float(wv.y & 0xffff0000u) - p.lr * v[3];
        }
        if constexpr (EPI == EPI_F32) {
          if (mok && nl_ < nvalid)
            *reinterpret_cast<float4*>(reinterpret_cast<float*>(p.C) + crow + n) = make_float4(v[0], v[1], v[2], v[3]);
        } else {
          pk[g][0] = f2bf2(v[0], v[1]);
          pk[g][1] = f2bf2(v[2], v[3]);
          if constexpr (EPI == EPI_BIAS_ACT) {
            float ac[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) ac[r] = act_fwd_fast(v[r], p.act);
            pa[g][0] = f2bf2(ac[0], ac[1]);
            pa[g][1] = f2bf2(ac[2], ac[3]);
          }
        }
      }
      if constexpr (EPI != EPI_F32) {
        // Lanes l and l + 32 hold the two 4-column halves of each 8-column group of one
        // row.  Swapping the upper lanes of group 2h with the lower lanes of group 2h+1
        // leaves lane l with columns 16h .. 16h+7 and lane l + 32 with 16h+8 .. 16h+15,
        // so each lane writes 16 contiguous bytes (all lanes take part in the swaps).
#pragma unroll
        for (int h2 = 0; h2 < 2; ++h2) {
#pragma unroll
          for (int q = 0; q < 2; ++q) {
            const auto r = __builtin_amdgcn_permlane32_swap(pk[2 * h2][q], pk[2 * h2 + 1][q], false, false);
            pk[2 * h2][q] = r[0];
            pk[2 * h2 + 1][q] = r[1];
            if constexpr (EPI == EPI_BIAS_ACT) {
              const auto ra = __builtin_amdgcn_permlane32_swap(pa[2 * h2][q], pa[2 * h2 + 1][q], false, false);
              pa[2 * h2][q] = ra[0];
              pa[2 * h2 + 1][q] = ra[1];
            }
          }
          const int c = cb + 16 * h2 + 8 * lhi;
          if (mok && c < nvalid) {
            *reinterpret_cast<uint4*>(reinterpret_cast<bf16*>(p.C) + crow + n0 + c) =
                make_uint4(pk[2 * h2][0], pk[2 * h2][1], pk[2 * h2 + 1][0], pk[2 * h2 + 1][1]);
            if constexpr (EPI == EPI_BIAS_ACT)
              *reinterpret_cast<uint4*>(reinterpret_cast<bf16*>(p.C2) + crow + n0 + c) =
                  make_uint4(pa[2 * h2][0], pa[2 * h2][1], pa[2 * h2 + 1][0], pa[2 * h2 + 1][1]);
          }
        }
      }
    };

    if constexpr (XB) {
      if (xl) {
        // the extra block's piece: rows BM .. BM+31 of the tile, column block wm
        const int ml = BM + l32;
        const bool mok = ml < mvalid;
        const int cb = wn * WTN + wm * 32;
        uint2 aux_x[4];
        if constexpr (HAS_AUX) {
          const int64_t arow = (int64_t)(off + m0 + (mok ? ml : 0)) * p.ldc;
#pragma unroll
          for (int g = 0; g < 4; ++g) {
            const int nl_ = cb + 8 * g + 4 * lhi;
            aux_x[g] = *reinterpret_cast<const uint2*>(p.aux + arow + n0 + (nl_ < nvalid ? nl_ : 0));
          }
        }
        emit_direct(accx, cb, (int64_t)(off + m0 + ml) * p.ldc, mok, bias_x, aux_x);
      }
    }
    if constexpr (SGD_SLOT) {
      // one piece: stage its accumulators, read them back in the store layout, update
      // and store (GUARD: some rows or columns of the tile are past the matrix); the
      // waits for the parameter loads are the compiler's, per register
      auto piece = [&](auto GUARDc, int pc, int buf) {
        constexpr bool GUARD = decltype(GUARDc)::value;
        const int j = pc / HP, h = pc % HP;
#pragma unroll
        for (int ii = 0; ii < 2; ++ii)
#pragma unroll
          for (int g = 0; g < 4; ++g) {
            const f32x16_t& a = acc[2 * h + ii][j];
            *reinterpret_cast<float4*>(s32 + s32_off(l32, ii * 8 + 2 * g + lhi)) =
                make_float4(a[4 * g], a[4 * g + 1], a[4 * g + 2], a[4 * g + 3]);
          }
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
        float v[4][8];
#pragma unroll
        for (int qd = 0; qd < 4; ++qd) {
          const int r = (lane >> 3) + 8 * qd, c8 = lane & 7;
          const float4 lo = *reinterpret_cast<const float4*>(s32 + s32_off(r, 2 * c8));
          const float4 hi = *reinterpret_cast<const float4*>(s32 + s32_off(r, 2 * c8 + 1));
          v[qd][0] = lo.x; v[qd][1] = lo.y; v[qd][2] = lo.z; v[qd][3] = lo.w;
          v[qd][4] = hi.x; v[qd][5] = hi.y; v[qd][6] = hi.z; v[qd][7] = hi.w;
        }
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
        const uint4 (&wv)[4] = wold[buf];
#pragma unroll
        for (int qd = 0; qd < 4; ++qd) {
          const uint32_t w4[4] = {wv[qd].x, wv[qd].y, wv[qd].z, wv[qd].w};
          uint32_t o[4];
#pragma unroll
          for (int q2 = 0; q2 < 4; ++q2) {
            const float a0 = __uint_as_float(w4[q2] << 16) - p.lr * v[qd][2 * q2];
            const float a1 = __uint_as_float(w4[q2] & 0xffff0000u) - p.lr * v[qd][2 * q2 + 1];
            o[q2] = f2bf2(a0, a1);
          }
          const int ml = (j * WM + wm) * 32 + (lane >> 3) + 8 * qd;
          const int col = wn * WTN + 64 * h + 8 * (lane & 7);
          if (!GUARD || (ml < mvalid && col < nvalid)) {
            uint4* dst = reinterpret_cast<uint4*>(W + (int64_t)e * p.c_gstride + (int64_t)(m0 + ml) * p.ldc + n0 + col);
            const uint4 ov = make_uint4(o[0], o[1], o[2], o[3]);
            if constexpr (STO == STORE_STAGED_NT) {
              typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
              __builtin_nontemporal_store(__builtin_bit_cast(u32x4_t, ov), reinterpret_cast<u32x4_t*>(dst));
            } else {
              *dst = ov;
            }
          }
        }
      };
      if (np == TM * HP && mvalid >= BM && nvalid >= BN) {
#pragma unroll
        for (int pc = 0; pc < TM * HP; ++pc) {
          if (pc == 0) load_piece(0, wold[0]);
          if (pc + 1 < TM * HP) load_piece(pc + 1, wold[(pc + 1) & 1]);
          piece(std::false_type{}, pc, pc & 1);
        }
      } else {
#pragma unroll
        for (int pc = 0; pc < TM * HP; ++pc) {
          if (pc < np) {
            load_piece(pc, wold[0]);
            piece(std::true_type{}, pc, 0);
          }
        }
      }
      // every wave is done with ring slot 1 before the next tile's stage 1 lands there
      block_sync_lds();
    }
#pragma unroll
    for (int j = 0; j < TM; ++j) {
      const int ml = (j * WM + wm) * 32 + l32;
      if (SGD_SLOT || j >= nl) continue;
      int64_t crow;
      if constexpr (GM == GROUP_M) crow = (int64_t)(off + m0 + ml) * p.ldc;
      else crow = (int64_t)e * p.c_gstride + (int64_t)(m0 + ml) * p.ldc;
      const bool mok = ml < mvalid;
      // this 32-row block of the tile read in C's layout (h for the activation
      // derivative; the parameters themselves for the SGD update), all loaded before
      // the block's first store (a load issued after a store also waits for the store)
      uint2 aux_v[HAS_AUX ? TN : 1][4];
      if constexpr (HAS_AUX) {
        const int mr = mok ? ml : 0;
        int64_t arow;
        if constexpr (GM == GROUP_M) arow = (int64_t)(off + m0 + mr) * p.ldc;
        else arow = (int64_t)e * p.c_gstride + (int64_t)(m0 + mr) * p.ldc;
        const bf16* src = EPI == EPI_SGD ? reinterpret_cast<const bf16*>(p.C) : p.aux;
#pragma unroll
        for (int i = 0; i < TN; ++i)
#pragma unroll
          for (int g = 0; g < 4; ++g) {
            const int nl_ = wn * WTN + i * 32 + 8 * g + 4 * lhi;
            aux_v[i][g] = *reinterpret_cast<const uint2*>(src + arow + n0 + (nl_ < nvalid ? nl_ : 0));
          }
      }
      if constexpr (STO != STORE_DIRECT) {
        // 64 output columns (two 32-column blocks) at a time through the wave's staging
        // area: lane (row l32, half lhi) writes its 4 x 8 bytes of each block, then lane
        // L reads row L/8 + 8q, chunk L%8, and stores the whole 128-byte line piece.
        char* stg = smem + STAGES * SBYTES + wave * STG_WAVE_BYTES;
        const int rb = (j * WM + wm) * 32;
        auto stage_out = [&](const uint32_t (&q)[2][4][2], bf16* out, int h) {
#pragma unroll
          for (int ii = 0; ii < 2; ++ii)
#pragma unroll
            for (int g = 0; g < 4; ++g)
              *reinterpret_cast<uint2*>(stg + stg_off(l32, 4 * ii + g) + lhi * 8) = make_uint2(q[ii][g][0], q[ii][g][1]);
          asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
#pragma unroll
          for (int qd = 0; qd < 4; ++qd) {
            const int r = (lane >> 3) + 8 * qd, c = lane & 7;
            const uint4 v = *reinterpret_cast<const uint4*>(stg + stg_off(r, c));
            const int ml = rb + r, col = wn * WTN + 64 * h + 8 * c;
            int64_t orow;
            if constexpr (GM == GROUP_M) orow = (int64_t)(off + m0 + ml) * p.ldc;
            else orow = (int64_t)e * p.c_gstride + (int64_t)(m0 + ml) * p.ldc;
            if (ml < mvalid && col < nvalid) {
              uint4* dst = reinterpret_cast<uint4*>(out + orow + n0 + col);
              if constexpr (STO == STORE_STAGED_NT) {
                typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
                __builtin_nontemporal_store(__builtin_bit_cast(u32x4_t, v), reinterpret_cast<u32x4_t*>(dst));
              } else {
                *dst = v;
              }
            }
          }
        };
#pragma unroll
        for (int h = 0; h < TN / 2; ++h) {
          uint32_t pk2[2][4][2], pa2[2][4][2];
#pragma unroll
          for (int ii = 0; ii < 2; ++ii) {
            const int i = 2 * h + ii;
#pragma unroll
            for (int g = 0; g < 4; ++g) {
              const int nl_ = wn * WTN + i * 32 + 8 * g + 4 * lhi;
              float v[4];
#pragma unroll
              for (int r = 0; r < 4; ++r) v[r] = acc[i][j][4 * g + r];
              if constexpr (HAS_BIAS) {
                const uint2 b = bias_v[i][g];
                v[0] += __uint_as_float(b.x << 16); v[1] += __uint_as_float(b.x & 0xffff0000u);
                v[2] += __uint_as_float(b.y << 16); v[3] += __uint_as_float(b.y & 0xffff0000u);
              }
              if constexpr (EPI == EPI_DACT) {
                const uint2 hv = aux_v[i][g];
                v[0] *= act_bwd_fast(__uint_as_float(hv.x << 16), p.act);
                v[1] *= act_bwd_fast(__uint_as_float(hv.x & 0xffff0000u), p.act);
                v[2] *= act_bwd_fast(__uint_as_float(hv.y << 16), p.act);
                v[3] *= act_bwd_fast(__uint_as_float(hv.y & 0xffff0000u), p.act);
              }
              if constexpr (EPI == EPI_SGD) {
                const uint2 wv = aux_v[i][g];
                v[0] = __uint_as_float(wv.x << 16) - p.lr * v[0];
                v[1] = __uint_as_float(wv.x & 0xffff0000u) - p.lr * v[1];
                v[2] = __uint_as_float(wv.y << 16) - p.lr * v[2];
                v[3] = __uint_as_float(wv.y & 0xffff0000u) - p.lr * v[3];
              }
              (void)nl_;
              pk2[ii][g][0] = f2bf2(v[0], v[1]);
              pk2[ii][g][1] = f2bf2(v[2], v[3]);
              if constexpr (EPI == EPI_BIAS_ACT) {
                float a[4];
#pragma unroll
                for (int r = 0; r < 4; ++r) a[r] = act_fwd_fast(v[r], p.act);
                pa2[ii][g][0] = f2bf2(a[0], a[1]);
                pa2[ii][g][1] = f2bf2(a[2], a[3]);
              }
            }
          }
          stage_out(pk2, reinterpret_cast<bf16*>(p.C), h);
          if constexpr (EPI == EPI_BIAS_ACT) stage_out(pa2, reinterpret_cast<bf16*>(p.C2), h);
        }
        continue;
      }
#pragma unroll
      for (int i = 0; i < TN; ++i)
        emit_direct(acc[i][j], wn * WTN + i * 32, crow, mok, bias_v[HAS_BIAS ? i : 0], aux_v[HAS_AUX ? i : 0]);
    }
    if constexpr (PRE < STAGES) {
      // stages issued after the epilogue: the stores are no longer the newest operations
      prev_stores = 0;
      if (more) {
#pragma unroll
        for (int st = PRE > early ? PRE : early; st < STAGES; ++st)
          if (st < nxt.nk) issue(nxt, st);
      }
    }
  }
}

template <int BM, int BN, int STAGES, bool A_T, bool B_T, int BK, int NW = 8, int STO = STORE_DIRECT, int XB = 0>
constexpr size_t gemm2_lds_bytes() {
  return (size_t)STAGES * (BM + (XB ? 32 : 0) + BN) * BK * 2 +
         (STO != STORE_DIRECT ? (size_t)NW * STG_WAVE_BYTES : 0);
}

}  // namespace dmoe
