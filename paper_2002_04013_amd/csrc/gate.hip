// Structured gate, exact TopK over the expert grid and Eq. 1 weights
// (Sec. 3.2, Eq. 1, App. C), plus the gate's backward pass.
#include <type_traits>

#include "common.hpp"
#include "gemm.hpp"
#include "gemm2.hpp"

namespace dmoe {

constexpr int GATE_TB = 32;     // tokens per block
constexpr int GATE_KC = 16;     // k chunk staged in LDS
constexpr int GATE_NT = 256;

struct GateArgs {
  const void* x; const void* Wg; const void* bg; const uint8_t* alive;
  int32_t* idx; float* w; float* g; float* scores;
  int T, D, d, M, k, dM, N;
};

// One token's selection from its fp64 gate scores s64[d*M] (Sec. 3.2, Eq. 1, App. C):
//  * decision scores are the fp32 roundings of the scores;
//  * per dimension, the best min(K1, M) indices by (score desc, index asc), kept in
//    registers by an insertion network (ties keep the earlier, lower index);
//  * the cells whose rank product is at most K1 (the only cells that can be among
//    the K1 best: a cell with per-dimension ranks r_i is beaten by the
//    prod(r_i + 1) - 1 cells taking an equal or better index in every dimension),
//    ranked by their fp64 total of d fp32 values in dimension order, ties to the
//    lower flat index;
//  * Eq. 1 weights over the chosen experts that are alive, from fp64 totals.
// When the nonzero scores span more than 2^26 in magnitude, an fp64 total of d fp32
// values may round and the dominance argument no longer holds exactly; then every
// cell of the grid is ranked.
// CERT (bf16 MFMA scores): K1 = k+1 cells (k if k = N) are ranked, and the selection
// is kept only if their totals are separated by more than 2E, E = d (delta_max +
// amax 2^-23) with delta = gam * ab[c] the bound on the score's accumulation error;
// the span must stay below 2^25.  Returns false (nothing written) otherwise.
// CAP: list capacity, at least K1 (the callers pick 5 when K1 <= 5, else KMAX + 1;
// for ALIVE 7 when k <= 4, else KMAX + 3).
// ALIVE (TopK among the alive experts, with CERT): the K1 = min(N, CAP) best cells are
// ranked the same way; walking them in order, the first k alive ones are the k best
// alive experts of the whole grid as soon as the k-th of them lies within those K1 (a
// cell outside the K1 best is beaten by all of them).  The selection is kept if the
// k-th alive cell is found there, the totals up to the cell after it are separated by
// more than 2E (or every cell was ranked), and the span condition holds; otherwise
// nothing is written (the token goes to the exact alive-first path).
template <bool CERT, int CAP, bool ALIVE = false>
__device__ __forceinline__ bool select_token_cap(const double* s64, const float* ab, const uint8_t* alive, int d,
                                                 int M, int k, int N, float gam, int32_t* idx_out, float* w_out,
                                                 float* g_out) {
  static_assert(!ALIVE || CERT, "alive-first selection on certified MFMA scores");
  const int K1 = ALIVE ? (N < CAP ? N : CAP) : (CERT && k < N ? k + 1 : k);
  const int L = K1 < M ? K1 : M;
  float lv[DMAX][CAP];
  int li[DMAX][CAP];
  float amax = 0.f, amin = 3.4e38f, dmax = 0.f;
#pragma unroll
  for (int i = 0; i < DMAX; ++i) {
#pragma unroll
    for (int p = 0; p < CAP; ++p) { lv[i][p] = -INFINITY; li[i][p] = 0; }
    if (i < d) {
      for (int u = 0; u < M; ++u) {
        float v = (float)s64[i * M + u];
        int id = u;
        const float av = fabsf(v);
        if (av > 0.f) { amax = fmaxf(amax, av); amin = fminf(amin, av); }
        if constexpr (CERT) dmax = fmaxf(dmax, gam * ab[i * M + u]);
#pragma unroll
        for (int p = 0; p < CAP; ++p) {
          const bool sw = v > lv[i][p];
          const float ov = lv[i][p];
          const int oi = li[i][p];
          lv[i][p] = sw ? v : ov; li[i][p] = sw ? id : oi;
          v = sw ? ov : v; id = sw ? oi : id;
        }
      }
    }
  }
  // top K1 cells: fp64 total, flat index, and the grid indices packed 8 bits per dim
  double tv[CAP];
  int tf[CAP], tu[CAP];
#pragma unroll
  for (int p = 0; p < CAP; ++p) { tv[p] = -INFINITY; tf[p] = 0x7fffffff; tu[p] = 0; }
  auto insert = [&](double v, int f, int uu) {
#pragma unroll
    for (int p = 0; p < CAP; ++p) {
      const bool sw = v > tv[p] || (v == tv[p] && f < tf[p]);
      const double ov = tv[p];
      const int of = tf[p], ou = tu[p];
      tv[p] = sw ? v : ov; tf[p] = sw ? f : of; tu[p] = sw ? uu : ou;
      v = sw ? ov : v; f = sw ? of : f; uu = sw ? ou : uu;
    }
  };
  const bool narrow = !(amax > 0.f) || amax <= amin * (CERT ? 33554432.f : 67108864.f);   // 2^25 / 2^26
  if (CERT && !narrow) return false;
  if (narrow) {
    // odometer over the rank digits r_0 .. r_{d-1} (last digit fastest), visiting only
    // the tuples with prod(r_i + 1) <= K1: a digit whose prefix product would exceed
    // K1 carries into the previous digit at once
    int r[DMAX];
#pragma unroll
    for (int i = 0; i < DMAX; ++i) r[i] = 0;
    for (int guard = 0; guard < 4096; ++guard) {
      int prod = 1;
#pragma unroll
      for (int i = 0; i < DMAX; ++i) if (i < d) prod *= r[i] + 1;
      if (prod <= K1) {
        double tot = 0.0;
        int flat = 0, uu = 0;
#pragma unroll
        for (int i = 0; i < DMAX; ++i) {
          if (i < d) {
            // element r[i] of the lists, by selects (the lists stay in registers)
            float pv = lv[i][0];
            int pi = li[i][0];
#pragma unroll
            for (int p = 1; p < CAP; ++p) { pv = r[i] == p ? lv[i][p] : pv; pi = r[i] == p ? li[i][p] : pi; }
            tot += (double)pv;
            flat = flat * M + pi;
            uu |= pi << (8 * i);
          }
        }
        insert(tot, flat, uu);
      }
      // next tuple: bump the last digit; a digit that reaches L, or makes the product
      // exceed K1 (so every larger value of it does too), resets and carries
      bool carry = true;
#pragma unroll
      for (int i = DMAX - 1; i >= 0; --i) {
        if (i < d && carry) {
          r[i] += 1;
          int pr = 1;
#pragma unroll
          for (int ii = 0; ii < DMAX; ++ii) if (ii < d) pr *= r[ii] + 1;
          if (r[i] >= L || pr > K1) r[i] = 0;
          else carry = false;
        }
      }
      if (carry) break;                  // every digit wrapped: done
    }
  } else {
    int u[DMAX];
#pragma unroll
    for (int i = 0; i < DMAX; ++i) u[i] = 0;
    for (int f = 0; f < N; ++f) {
      double tot = 0.0;
      int uu = 0;
#pragma unroll
      for (int i = 0; i < DMAX; ++i) if (i < d) { tot += (double)(float)s64[i * M + u[i]]; uu |= u[i] << (8 * i); }
      insert(tot, f, uu);
#pragma unroll
      for (int i = DMAX - 1; i >= 0; --i) {        // next flat index: last dim fastest
        if (i < d) {
          if (++u[i] < M) break;
          u[i] = 0;
        }
      }
    }
  }
  if constexpr (ALIVE) {
    // the first k alive cells among the K1 best; position of the k-th
    int pk = -1, cnt = 0;
#pragma unroll
    for (int p = 0; p < CAP; ++p) {
      const bool live = p < K1 && cnt < k && (alive == nullptr || alive[tf[p]] != 0);
      if (live) {
        ++cnt;
        if (cnt == k) pk = p;
      }
    }
    if (pk < 0) return false;
    if (pk + 1 >= K1 && K1 < N) return false;      // the cell after the k-th is not ranked
    const double E = (double)d * ((double)dmax + (double)amax * 1.1920928955078125e-7);
    bool sep = true;
#pragma unroll
    for (int j = 0; j + 1 < CAP; ++j)
      if (j <= pk && j + 1 < K1) sep = sep && (tv[j] - tv[j + 1] > 2.0 * E);
    if (!sep) return false;
    // keep only the alive cells, in order: compact positions 0 .. pk
    int w = 0;
#pragma unroll
    for (int p = 0; p < CAP; ++p) {
      if (p <= pk && (alive == nullptr || alive[tf[p]] != 0)) {
        // move entry p to slot w (w <= p): selects over the register arrays
        const double vv = tv[p];
        const int ff = tf[p], uu = tu[p];
#pragma unroll
        for (int q = 0; q < CAP; ++q)
          if (q == w) { tv[q] = vv; tf[q] = ff; tu[q] = uu; }
        ++w;
      }
    }
  } else if constexpr (CERT) {
    const double E = (double)d * ((double)dmax + (double)amax * 1.1920928955078125e-7);
    bool sep = true;
#pragma unroll
    for (int j = 0; j + 1 < CAP; ++j)
      if (j + 1 < K1) sep = sep && (tv[j] - tv[j + 1] > 2.0 * E);
    if (!sep) return false;
  }
  // Eq. 1 weights from the fp64 totals of the chosen experts, over the alive ones
  constexpr int KJ = CAP < KMAX ? CAP : KMAX;      // k <= K1 <= CAP
  double gx[KJ];
  bool live[KJ];
#pragma unroll
  for (int j = 0; j < KJ; ++j) live[j] = j < k && (alive == nullptr || alive[tf[j]] != 0);
  double m = -1.0e308;
  bool any = false;
#pragma unroll
  for (int j = 0; j < KJ; ++j) {
    gx[j] = 0.0;
    if (j < k) {
      double t = 0.0;
#pragma unroll
      for (int i = 0; i < DMAX; ++i) if (i < d) t += s64[i * M + ((tu[j] >> (8 * i)) & 0xff)];
      gx[j] = t;
      if (live[j]) { any = true; m = t > m ? t : m; }
    }
  }
  float ex[KJ];
  float sum = 0.f;
#pragma unroll
  for (int j = 0; j < KJ; ++j) {
    ex[j] = live[j] ? expf((float)(gx[j] - m)) : 0.f;
    sum += ex[j];
  }
#pragma unroll
  for (int j = 0; j < KJ; ++j) {
    if (j < k) {
      idx_out[j] = tf[j];
      w_out[j] = any ? ex[j] / sum : 0.f;
      if (g_out) g_out[j] = (float)gx[j];
    }
  }
  return true;
}

template <bool CERT, bool ALIVE = false>
__device__ __forceinline__ bool select_token(const double* s64, const float* ab, const uint8_t* alive, int d, int M,
                                             int k, int N, float gam, int32_t* idx_out, float* w_out, float* g_out) {
  if constexpr (ALIVE) {      // k + 3 cells ranked: up to two dead ones ahead of the k-th alive
    if (k <= 4) return select_token_cap<true, 7, true>(s64, ab, alive, d, M, k, N, gam, idx_out, w_out, g_out);
    return select_token_cap<true, KMAX + 3, true>(s64, ab, alive, d, M, k, N, gam, idx_out, w_out, g_out);
  }
  const int K1 = CERT && k < N ? k + 1 : k;
  if (K1 <= 5) return select_token_cap<CERT, 5>(s64, ab, alive, d, M, k, N, gam, idx_out, w_out, g_out);
  return select_token_cap<CERT, KMAX + 1>(s64, ab, alive, d, M, k, N, gam, idx_out, w_out, g_out);
}

template <typename E>
__global__ void __launch_bounds__(GATE_NT) gate_topk_kernel(GateArgs a) {
  extern __shared__ __align__(16) unsigned char sm[];
  const int dM = a.dM;
  double* xs = reinterpret_cast<double*>(sm);                         // [TB][KC]
  double* wsT = xs + GATE_TB * GATE_KC;                               // [KC][dM]
  double* s64 = wsT + GATE_KC * dM;                                   // [TB][dM + 1]

  const int tid = threadIdx.x;
  const int t0 = blockIdx.x * GATE_TB;
  const E* x = reinterpret_cast<const E*>(a.x);
  const E* W = reinterpret_cast<const E*>(a.Wg);
  constexpr int TG = GATE_TB / 8;            // token groups of 8
  const int items = dM * TG;                 // (column, token group) work items
  constexpr int IPT = DM_MAX * TG / GATE_NT;
  double acc[IPT][8];
#pragma unroll
  for (int it = 0; it < IPT; ++it)
#pragma unroll
    for (int r = 0; r < 8; ++r) acc[it][r] = 0.0;

  for (int k0 = 0; k0 < a.D; k0 += GATE_KC) {
    for (int q = tid; q < GATE_TB * GATE_KC; q += GATE_NT) {
      const int tt = q / GATE_KC, kk = q % GATE_KC;
      const int t = t0 + tt;
      xs[q] = t < a.T ? (double)ldf(x + (int64_t)t * a.D + k0 + kk) : 0.0;
    }
    for (int q = tid; q < GATE_KC * dM; q += GATE_NT) {
      const int c = q / GATE_KC, kk = q % GATE_KC;
      wsT[kk * dM + c] = (double)ldf(W + (int64_t)c * a.D + k0 + kk);
    }
    __syncthreads();
#pragma unroll
    for (int it = 0; it < IPT; ++it) {
      const int item = tid + it * GATE_NT;
      if (item < items) {
        const int c = item % dM, tg = item / dM;
        for (int kk = 0; kk < GATE_KC; ++kk) {
          const double wv = wsT[kk * dM + c];
#pragma unroll
          for (int r = 0; r < 8; ++r) acc[it][r] = fma(xs[(tg * 8 + r) * GATE_KC + kk], wv, acc[it][r]);
        }
      }
    }
    __syncthreads();
  }
#pragma unroll
  for (int it = 0; it < IPT; ++it) {
    const int item = tid + it * GATE_NT;
    if (item < items) {
      const int c = item % dM, tg = item / dM;
      const double b = a.bg ? (double)ldf(reinterpret_cast<const E*>(a.bg) + c) : 0.0;
#pragma unroll
      for (int r = 0; r < 8; ++r) {
        const double v = acc[it][r] + b;
        const int tt = tg * 8 + r;
        s64[tt * (dM + 1) + c] = v;
      }
    }
  }
  __syncthreads();
  if (a.scores) {
    for (int q = tid; q < GATE_TB * dM; q += GATE_NT) {
      const int t = t0 + q / dM;
      if (t < a.T) a.scores[(int64_t)t * dM + q % dM] = (float)s64[(q / dM) * (dM + 1) + q % dM];
    }
  }
  if (tid < GATE_TB && t0 + tid < a.T) {
    const int t = t0 + tid;
    select_token<false>(s64 + tid * (dM + 1), nullptr, a.alive, a.d, a.M, a.k, a.N, 0.f,
                        a.idx + (int64_t)t * a.k, a.w + (int64_t)t * a.k, a.g ? a.g + (int64_t)t * a.k : nullptr);
  }
}

// ---------------------------------------------------------------- bf16: MFMA scores + certificate
//
// Scores are computed on bf16 MFMA: products of bf16 values are exact in fp32, 32 of
// them are summed per MFMA chunk pair in fp32, and the chunk sums are added in fp64.
// A second MFMA over |x|.|w| gives A = sum_k |x_k w_k|, which bounds the accumulation
// error of each score:  |S - exact| <= delta = (gamma_32 + (D/32 + 8) 2^-52) A,
// gamma_n = n u / (1 - n u) with u = 2^-23 (no assumption about the MFMA's internal
// rounding beyond single-precision operations, directed rounding included).  Decision
// scores of the GPU and of an exact computation then differ by at most delta + 1 ulp
// each, a cell total by at most d (delta + ulp) =: E.  If the k+1 best cells (k when
// k = N) are separated by gaps larger than 2E, the exact scores give the same TopK in
// the same order; such tokens are certified.  The others are appended to a device
// queue and recomputed with exact fp64 accumulation by gate_exact_kernel.

constexpr int GM_TOK = 32;        // tokens per block (one MFMA row block)
constexpr int GM_RING = 2;        // x groups (32 tokens x 64 d_model, 4 KB) in flight per wave
// Waves per block (each a share of the d_model groups): 2 from d_model 2048 on, else 1.
// A 2-slot ring keeps a block's LDS small (8 KB per slot and wave with 32 gate columns),
// so that several blocks share a compute unit and one block's selection overlaps the
// others' loads.
constexpr int gm_kw(int64_t D) { return D >= 2048 ? 2 : 1; }
constexpr int GX_NT = 512;        // exact recomputation: threads per token

struct GateMfmaArgs {
  GateArgs a;
  int flags;
  float gam;                       // gamma_32 + (D/32+8) 2^-52, times 1/(1 - gamma_D)
  int32_t* queue;                  // [0] count, [GQ_HEAD + i] token ids
};

__device__ __forceinline__ void g2l16(const void* g, void* lds_wave_base) {
  __builtin_amdgcn_global_load_lds((__attribute__((address_space(1))) void*)g,
                                   (__attribute__((address_space(3))) void*)lds_wave_base, 16, 0, 0);
}

// A block of KW waves scores 32 tokens against all d*M gate columns; wave w takes
// the d_model groups w, w + KW, ... (groups of 64 values).  x and Wg stream
// through a per-wave LDS ring of GM_RING groups (direct global->LDS loads, 8 rows x
// 128 bytes per instruction, 16-byte chunks XOR-swizzled by row): a slot holds 32
// token rows, then 32*CB gate-column rows.  Within a group, lane half h holds
// d_model offsets 32h .. 32h+31 and MFMA chunk j takes 32h+8j .. 32h+8j+7 from both
// operands (the contraction order is permuted identically for x and Wg).  The
// waves' fp64 partial sums are added in wave order in LDS, then one lane per token
// selects.
// ALIVE: TopK among the alive experts (the certified selection extended until k alive
// cells are decided; see select_token_cap).
template <int CB, int KW, bool ALIVE = false>   // 32-column blocks of the d*M gate columns; waves
__global__ void __launch_bounds__(64 * KW) gate_topk_mfma(GateMfmaArgs ga) {
  const GateArgs& a = ga.a;
  extern __shared__ __align__(1024) unsigned char sm[];
  constexpr int SLOT = 4096 * (1 + CB);          // bytes per ring slot
  constexpr int LPG = 4 * (1 + CB);              // load instructions per group
  const int dM = a.dM;
  const int lane = threadIdx.x & 63;
  const int wv = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int t0 = blockIdx.x * GM_TOK;
  const bool exact_all = (ga.flags & DMOE_FLAG_GATE_EXACT) != 0;
  if (exact_all) {                       // every token goes to the exact path
    if (threadIdx.x < GM_TOK && t0 + threadIdx.x < a.T)
      ga.queue[GQ_HEAD + atomicAdd(ga.queue, 1)] = t0 + threadIdx.x;
    return;
  }
  const bf16* x = reinterpret_cast<const bf16*>(a.x);
  const bf16* W = reinterpret_cast<const bf16*>(a.Wg);
  const bf16* bg = reinterpret_cast<const bf16*>(a.bg);
  const int tok = lane & 31, half = lane >> 5;
  const int NG = a.D / 64;
  const int ng = NG > wv ? (NG - wv + KW - 1) / KW : 0;         // groups of this wave
  char* ring = reinterpret_cast<char*>(sm) + wv * (GM_RING * SLOT);
  // instruction q fills rows 8q .. 8q+7 of the slot (q < 4: tokens, then gate columns);
  // lane -> row 8q + lane/8, chunk lane%8 stored at position (lane%8) ^ (row%8)
  const int lrow = lane >> 3, lch = lane & 7;
  auto issue = [&](int m) {                       // the wave's m-th group
    char* slot = ring + (m % GM_RING) * SLOT;
    const int64_t k0 = (int64_t)64 * (wv + KW * m);
#pragma unroll
    for (int q = 0; q < 4 * (1 + CB); ++q) {
      const int r = 8 * q + lrow;
      const int c = lch ^ (r & 7);
      const bf16* src;
      if (q < 4) src = x + (int64_t)min(t0 + r, a.T - 1) * a.D;
      else src = W + (int64_t)min(r - 32, dM - 1) * a.D;
      g2l16(src + k0 + 8 * c, slot + q * 1024);
    }
  };
  // fragment of slot row `row`, chunk 4*half + jj
  auto frag = [&](int m, int row, int jj) {
    const char* slot = ring + (m % GM_RING) * SLOT;
    const int c = (4 * half + jj) ^ (row & 7);
    return *reinterpret_cast<const bf16x8_t*>(slot + row * 128 + c * 16);
  };
#pragma unroll
  for (int m = 0; m < GM_RING; ++m)
    if (m < ng) issue(m);

  double acc[CB][16];
  f32x16_t aacc[CB];
#pragma unroll
  for (int cb = 0; cb < CB; ++cb)
#pragma unroll
    for (int r = 0; r < 16; ++r) { acc[cb][r] = 0.0; aacc[cb][r] = 0.f; }
  for (int m = 0; m < ng; ++m) {
    // Vector-memory operations retire in issue order, and group m is followed by the
    // groups issued after it, LPG loads each: once at most that many are
    // outstanding, group m has landed.
    static_assert(GM_RING == 2, "one group in flight behind the current one");
    if (m + 1 < ng) wait_vmcnt<LPG>(); else wait_vmcnt<0>();
    f32x16_t c[CB];
#pragma unroll
    for (int cb = 0; cb < CB; ++cb)
#pragma unroll
      for (int r = 0; r < 16; ++r) c[cb][r] = 0.f;
#pragma unroll
    for (int jj = 0; jj < 4; ++jj) {
      const bf16x8_t xq = frag(m, tok, jj);
      const uint4 xu = __builtin_bit_cast(uint4, xq);
      const uint4 xa = make_uint4(xu.x & 0x7fff7fffu, xu.y & 0x7fff7fffu, xu.z & 0x7fff7fffu, xu.w & 0x7fff7fffu);
#pragma unroll
      for (int cb = 0; cb < CB; ++cb) {
        const bf16x8_t wq = frag(m, 32 + 32 * cb + tok, jj);
        const uint4 wu = __builtin_bit_cast(uint4, wq);
        const uint4 wa = make_uint4(wu.x & 0x7fff7fffu, wu.y & 0x7fff7fffu, wu.z & 0x7fff7fffu, wu.w & 0x7fff7fffu);
        c[cb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wq, xq, c[cb], 0, 0, 0);
        aacc[cb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, wa),
                                                          __builtin_bit_cast(bf16x8_t, xa), aacc[cb], 0, 0, 0);
      }
      if (jj & 1) {                      // every 32 products the fp32 sums move to fp64
#pragma unroll
        for (int cb = 0; cb < CB; ++cb)
#pragma unroll
          for (int r = 0; r < 16; ++r) { acc[cb][r] += (double)c[cb][r]; c[cb][r] = 0.f; }
      }
    }
    // every lane has read group m from its slot (the wave's LDS reads retire in order
    // before the refill is issued); refill it with group m + RING
    __builtin_amdgcn_s_waitcnt(0xc07f);  // lgkmcnt(0), vmcnt/expcnt untouched
    asm volatile("" ::: "memory");
    if (m + GM_RING < ng) issue(m + GM_RING);
  }

  // partial sums to LDS in wave order (rows padded to an odd word count: distinct
  // banks per token), then one lane per token selects
  wait_vmcnt<0>();
  __syncthreads();                       // both rings drained before their memory is reused
  const int SLD = dM + 1;
  double* s64 = reinterpret_cast<double*>(sm);                 // [32][SLD]
  float* ab = reinterpret_cast<float*>(s64 + GM_TOK * SLD);    // [32][SLD]
  for (int w = 0; w < KW; ++w) {
    if (wv == w) {
#pragma unroll
      for (int cb = 0; cb < CB; ++cb) {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int cc = cb * 32 + 8 * (r >> 2) + 4 * half + (r & 3);
          if (cc < dM) {
            if (w == 0) {
              s64[tok * SLD + cc] = acc[cb][r] + (bg ? (double)bf2f(bg[cc]) : 0.0);
              ab[tok * SLD + cc] = aacc[cb][r];
            } else {
              s64[tok * SLD + cc] += acc[cb][r];
              ab[tok * SLD + cc] += aacc[cb][r];
            }
          }
        }
      }
    }
    __syncthreads();
  }
  if (threadIdx.x < GM_TOK && t0 + (int)threadIdx.x < a.T) {
    const int t = t0 + threadIdx.x;
    const bool ok = select_token<true, ALIVE>(s64 + lane * SLD, ab + lane * SLD, a.alive, a.d, a.M, a.k, a.N, ga.gam,
                                       a.idx + (int64_t)t * a.k, a.w + (int64_t)t * a.k,
                                       a.g ? a.g + (int64_t)t * a.k : nullptr);
    if (!ok) ga.queue[GQ_HEAD + atomicAdd(ga.queue, 1)] = t;
    if (ok && a.scores)
      for (int c = 0; c < dM; ++c) a.scores[(int64_t)t * dM + c] = (float)s64[lane * SLD + c];
  }
}

// Order-preserving 64-bit image of an fp64 value (larger value, larger key; no NaN).
__device__ __forceinline__ uint64_t ord64(double v) {
  const uint64_t b = (uint64_t)__double_as_longlong(v);
  return (b >> 63) ? ~b : (b | 0x8000000000000000ull);
}
// Cell keys (live, total, ~flat) compared lexicographically: alive first (when ranked
// that way), then the larger total, then the lower flat index (larger ~flat).
__device__ __forceinline__ bool cell_gt(uint32_t al, uint64_t at, uint32_t an, uint32_t bl, uint64_t bt,
                                        uint32_t bn) {
  return (al > bl) | ((al == bl) & ((at > bt) | ((at == bt) & (an > bn))));
}

// Exact path for the queued tokens: fp64 scores S[c] = sum_k x_k W[c][k] + b[c], then the
// selection.  Persistent blocks over the queue; a pass takes TB tokens: GX_TB = 8 where
// every token is queued (alive-first TopK, or exact scores asked for: the tokens of a
// pass share each load of Wg, and one wave selects for each), 1 for the few tokens the
// certificate rejects (lowest latency, two blocks per compute unit).  Wave w owns the gate columns
// [w cpw, (w+1) cpw), cpw = ceil(dM / 8), GX_CT at a time; lane l sums the 16-byte
// vectors l, l + 64, ... of the rows (each wave load is 1 KB of one row) with fp64
// FMAs of the exact element values, P vectors' loads issued before any is used; a
// shuffle tree adds the 64 lane sums.
constexpr int GX_CT = 4;          // gate columns per wave pass of the exact scores
constexpr int GX_TB = 8;          // tokens per pass when every token is queued (one per wave)

// Element q (compile-time after unrolling) of a 16-byte vector, as a float.
template <typename E> __device__ __forceinline__ float vec_elem(const uint4& v, int q);
template <> __device__ __forceinline__ float vec_elem<float>(const uint4& v, int q) {
  return __uint_as_float(q == 0 ? v.x : q == 1 ? v.y : q == 2 ? v.z : v.w);
}
template <> __device__ __forceinline__ float vec_elem<bf16>(const uint4& v, int q) {
  const uint32_t w = (q >> 1) == 0 ? v.x : (q >> 1) == 1 ? v.y : (q >> 1) == 2 ? v.z : v.w;
  return __uint_as_float((q & 1) ? (w & 0xffff0000u) : (w << 16));
}

template <typename E, int TB, int P>
__device__ __forceinline__ void exact_scores(const GateArgs& a, const int* tok, double (*s64)[DM_MAX]) {
  constexpr int VEC = 16 / sizeof(E);
  constexpr int NW = GX_NT / 64;
  const int lane = threadIdx.x & 63;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int cpw = (a.dM + NW - 1) / NW;
  const int cend = min(a.dM, (w + 1) * cpw);
  const int nv = a.D / VEC;
  const E* x = reinterpret_cast<const E*>(a.x);
  const E* W = reinterpret_cast<const E*>(a.Wg);
  const E* bg = reinterpret_cast<const E*>(a.bg);
  for (int c0 = w * cpw; c0 < cend; c0 += GX_CT) {
    const E* wr[GX_CT];
    const E* xr[TB];
#pragma unroll
    for (int c = 0; c < GX_CT; ++c) wr[c] = W + (int64_t)min(c0 + c, a.dM - 1) * a.D;
#pragma unroll
    for (int t = 0; t < TB; ++t) xr[t] = x + (int64_t)tok[t] * a.D;
    double acc[TB][GX_CT];
#pragma unroll
    for (int t = 0; t < TB; ++t)
#pragma unroll
      for (int c = 0; c < GX_CT; ++c) acc[t][c] = 0.0;
    for (int v0 = lane; v0 < nv; v0 += 64 * P) {
      uint4 wv[P][GX_CT], xv[P][TB];
#pragma unroll
      for (int p = 0; p < P; ++p) {
        const int64_t v = v0 + 64 * p;
        if (v < nv) {
#pragma unroll
          for (int c = 0; c < GX_CT; ++c) wv[p][c] = *reinterpret_cast<const uint4*>(wr[c] + v * VEC);
#pragma unroll
          for (int t = 0; t < TB; ++t) xv[p][t] = *reinterpret_cast<const uint4*>(xr[t] + v * VEC);
        }
      }
#pragma unroll
      for (int p = 0; p < P; ++p) {
        if (v0 + 64 * p < nv) {
#pragma unroll
          for (int q = 0; q < VEC; ++q) {
            double xd[TB], wd[GX_CT];
#pragma unroll
            for (int t = 0; t < TB; ++t) xd[t] = (double)vec_elem<E>(xv[p][t], q);
#pragma unroll
            for (int c = 0; c < GX_CT; ++c) wd[c] = (double)vec_elem<E>(wv[p][c], q);
#pragma unroll
            for (int t = 0; t < TB; ++t)
#pragma unroll
              for (int c = 0; c < GX_CT; ++c) acc[t][c] = fma(xd[t], wd[c], acc[t][c]);
          }
        }
      }
    }
#pragma unroll
    for (int t = 0; t < TB; ++t) {
#pragma unroll
      for (int c = 0; c < GX_CT; ++c) {
        double v = acc[t][c];
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
        if (lane == 0 && c0 + c < cend) s64[t][c0 + c] = v + (bg ? (double)ldf(bg + c0 + c) : 0.0);
      }
    }
  }
}

// Cell key (live, ord64(total), ~flat): the lexicographic maximum is the best cell.
struct CellKey { uint32_t l; uint64_t t; uint32_t n; };

__device__ __forceinline__ bool key_gt(const CellKey& a, const CellKey& b) {
  return cell_gt(a.l, a.t, a.n, b.l, b.t, b.n);
}
__device__ __forceinline__ CellKey key_sel(bool c, const CellKey& a, const CellKey& b) {
  return CellKey{c ? a.l : b.l, c ? a.t : b.t, c ? a.n : b.n};
}

template <int CTRL, int ROWS>
__device__ __forceinline__ uint64_t u64_max_dpp(uint64_t v) {
  const uint32_t lo = (uint32_t)__builtin_amdgcn_update_dpp((int)(uint32_t)v, (int)(uint32_t)v, CTRL, ROWS, 0xf, false);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_update_dpp((int)(uint32_t)(v >> 32), (int)(uint32_t)(v >> 32), CTRL,
                                                            ROWS, 0xf, false);
  const uint64_t o = ((uint64_t)hi << 32) | lo;
  return o > v ? o : v;
}

// Maximum of a 64-bit value over the wave (every lane gets it): within each row of 16
// lanes by DPP exchanges (lane i with i^1, i^2, 7-i, 15-i), then row r-1's last lane into
// row r (rows 1 and 3) and lane 31 into rows 2 and 3, so that lane 63 holds the maximum.
__device__ __forceinline__ uint64_t wave_max_u64(uint64_t v) {
  v = u64_max_dpp<0xB1, 0xf>(v);       // quad_perm [1,0,3,2]
  v = u64_max_dpp<0x4E, 0xf>(v);       // quad_perm [2,3,0,1]
  v = u64_max_dpp<0x141, 0xf>(v);      // row_half_mirror
  v = u64_max_dpp<0x140, 0xf>(v);      // row_mirror
  v = u64_max_dpp<0x142, 0xa>(v);      // row_bcast:15
  v = u64_max_dpp<0x143, 0xc>(v);      // row_bcast:31
  return ((uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(v >> 32), 63) << 32) |
         (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, 63);
}

// TopK by its definition for one token, by one wave: every cell of the grid is ranked by
// (alive first when ALIVE, total desc, flat asc), the totals adding the d fp32 decision
// scores sd (as fp64) in fp64 in dimension order.  Lane l scans the cells l, l + 64, ...
// (mixed-radix digits advanced by 64 per cell, four cells per step) into its own sorted
// list of the LK >= k best, then k rounds take the best list head of the wave: the
// largest live flag, then the largest total among those heads, ties to the larger
// ~flat; the owner drops it.  Eq. 1 weights over the chosen experts that are alive;
// lane j writes entry j.
template <bool ALIVE, int LK>
__device__ __forceinline__ void exact_select_wave(const GateArgs& a, const double* sc, const double* sd,
                                                  const uint8_t* alv, int t) {
  const int lane = threadIdx.x & 63;
  const int d = a.d, M = a.M, k = a.k, N = a.N;
  const CellKey none{0u, 0ull, 0u};                                 // below every real key
  CellKey L[LK];
#pragma unroll
  for (int j = 0; j < LK; ++j) L[j] = none;
  int u[DMAX], st[DMAX];
  {
    int rl = lane, rs = 64;
#pragma unroll
    for (int i = DMAX - 1; i >= 0; --i) {
      u[i] = 0; st[i] = 0;
      if (i < d) { u[i] = rl % M; rl /= M; st[i] = rs % M; rs /= M; }
    }
  }
  for (int f0 = lane; f0 < N; f0 += 4 * 64) {
    CellKey c[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const int f = f0 + 64 * q;
      double tot = 0.0;
#pragma unroll
      for (int i = 0; i < DMAX; ++i) if (i < d) tot += sd[i * M + u[i]];   // digits stay in [0, M)
      const uint32_t live = !ALIVE || alv[min(f, N - 1)] != 0 ? 1u : 0u;
      c[q] = key_sel(f < N, CellKey{live, ord64(tot + 0.0), ~(uint32_t)f}, none);   // -0 and +0 are one value
      int carry = 0;                                                  // digits of f + 64
#pragma unroll
      for (int i = DMAX - 1; i >= 0; --i) {
        if (i < d) {
          u[i] += st[i] + carry;
          carry = u[i] >= M;
          u[i] -= carry ? M : 0;
        }
      }
    }
#pragma unroll
    for (int q = 0; q < 4; ++q) {                                     // sorted insertion, no branches
      CellKey cur = c[q];
      bool go = false;
#pragma unroll
      for (int j = 0; j < LK; ++j) {
        const bool gt = go || key_gt(cur, L[j]);
        const CellKey old = L[j];
        L[j] = key_sel(gt, cur, old);
        cur = key_sel(gt, old, cur);
        go = gt;
      }
    }
  }
  int chosen[KMAX];
#pragma unroll
  for (int r = 0; r < KMAX; ++r) {
    chosen[r] = 0;
    if (r < k) {
      const CellKey h = L[0];
      uint32_t lmax = 1u;
      if (ALIVE) lmax = __ballot(h.l != 0u) != 0ull ? 1u : 0u;
      const uint64_t tt = h.l == lmax ? h.t : 0ull;                  // real totals have keys > 0
      const uint64_t tmax = wave_max_u64(tt);
      const uint64_t mask = __ballot(tt == tmax && h.l == lmax);
      int wl;
      if (__popcll(mask) == 1) {
        wl = __ffsll((unsigned long long)mask) - 1;
      } else {                                                       // equal totals: larger ~flat
        const uint64_t nn = (mask >> lane) & 1ull ? (uint64_t)h.n : 0ull;
        const uint64_t nmax = wave_max_u64(nn);
        wl = __ffsll((unsigned long long)__ballot(nn == nmax && ((mask >> lane) & 1ull))) - 1;
      }
      wl = __builtin_amdgcn_readfirstlane(wl);
      chosen[r] = (int)~(uint32_t)__builtin_amdgcn_readlane((int)h.n, wl);
      const bool pop = lane == wl;
#pragma unroll
      for (int j = 0; j < LK - 1; ++j) L[j] = key_sel(pop, L[j + 1], L[j]);
      L[LK - 1] = key_sel(pop, none, L[LK - 1]);
    }
  }
  // Eq. 1 weights from the fp64 totals of the chosen experts, over the alive ones
  // (uniform over the wave; lane j stores entry j)
  double gx[KMAX];
  bool lv[KMAX];
  double m = -1.0e308;
  bool any = false;
#pragma unroll
  for (int j = 0; j < KMAX; ++j) {
    gx[j] = 0.0;
    lv[j] = false;
    if (j < k) {
      int rem = chosen[j], v[DMAX];
#pragma unroll
      for (int i = DMAX - 1; i >= 0; --i) { v[i] = 0; if (i < d) { v[i] = rem % M; rem /= M; } }
      double tt = 0.0;
#pragma unroll
      for (int i = 0; i < DMAX; ++i) if (i < d) tt += sc[i * M + v[i]];
      gx[j] = tt;
      lv[j] = a.alive == nullptr || a.alive[chosen[j]] != 0;
      if (lv[j]) { any = true; m = tt > m ? tt : m; }
    }
  }
  float ex[KMAX];
  float sum = 0.f;
#pragma unroll
  for (int j = 0; j < KMAX; ++j) {
    ex[j] = lv[j] ? expf((float)(gx[j] - m)) : 0.f;
    sum += ex[j];
  }
  int my_idx = 0;
  float my_w = 0.f, my_g = 0.f;
#pragma unroll
  for (int j = 0; j < KMAX; ++j) {
    if (lane == j) { my_idx = chosen[j]; my_w = any ? ex[j] / sum : 0.f; my_g = (float)gx[j]; }
  }
  if (lane < k) {
    a.idx[(int64_t)t * k + lane] = my_idx;
    a.w[(int64_t)t * k + lane] = my_w;
    if (a.g) a.g[(int64_t)t * k + lane] = my_g;
  }
  if (a.scores)
    for (int c = lane; c < a.dM; c += 64) a.scores[(int64_t)t * a.dM + c] = (float)sc[c];
}

template <typename E, bool ALIVE, int TB, int P>
__device__ __forceinline__ void exact_pass(const GateArgs& a, const int32_t* queue, int n, int qg,
                                           double (*s64)[DM_MAX], double (*sd)[DM_MAX], const uint8_t* alv) {
  const int nt = min(TB, n - qg * TB);
  int tok[TB];
#pragma unroll
  for (int j = 0; j < TB; ++j) tok[j] = queue[GQ_HEAD + qg * TB + min(j, nt - 1)];   // pads repeat a token
  exact_scores<E, TB, P>(a, tok, s64);
  __syncthreads();
  for (int q = threadIdx.x; q < nt * a.dM; q += GX_NT)
    sd[q / a.dM][q % a.dM] = (double)(float)s64[q / a.dM][q % a.dM];
  __syncthreads();
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  if (w < nt) {
    if (a.k <= 4) exact_select_wave<ALIVE, 4>(a, s64[w], sd[w], alv, tok[w]);
    else exact_select_wave<ALIVE, KMAX>(a, s64[w], sd[w], alv, tok[w]);
  }
  __syncthreads();                                                   // s64, sd reused by the next pass
}

template <typename E, bool ALIVE, int TB>
__device__ __forceinline__ void exact_body(const GateArgs& a, const int32_t* queue, double (*s64)[DM_MAX],
                                           double (*sd)[DM_MAX], uint8_t* alv) {
  const int n = queue[0];
  const int ngrp = (n + TB - 1) / TB;
  if ((int)blockIdx.x >= ngrp) return;
  if (ALIVE) {
    for (int f = threadIdx.x; f < a.N; f += GX_NT) alv[f] = a.alive == nullptr || a.alive[f] != 0 ? 1 : 0;
    __syncthreads();
  }
  for (int qg = blockIdx.x; qg < ngrp; qg += gridDim.x)
    exact_pass<E, ALIVE, TB, TB == 1 ? 3 : 2>(a, queue, n, qg, s64, sd, alv);
}

// Every token queued (alive-first TopK, or exact scores asked for): GX_TB tokens a pass.
template <typename E, bool ALIVE>
__global__ void __launch_bounds__(GX_NT) gate_exact_kernel(GateArgs a, const int32_t* queue) {
  __shared__ double s64[GX_TB][DM_MAX];
  __shared__ double sd[GX_TB][DM_MAX];
  __shared__ uint8_t alv[ALIVE ? NMAX : 1];                          // alive flags (ALIVE ranking)
  exact_body<E, ALIVE, GX_TB>(a, queue, s64, sd, alv);
}

// The tokens the certificate rejects (bf16 MFMA scores): one token a pass, two blocks
// per compute unit.  ALIVE: ranked alive first.
template <bool ALIVE>
__global__ void __launch_bounds__(GX_NT) __attribute__((amdgpu_waves_per_eu(4)))
gate_exact_sparse_kernel(GateArgs a, const int32_t* queue) {
  __shared__ double s64[1][DM_MAX];
  __shared__ double sd[1][DM_MAX];
  __shared__ uint8_t alv[ALIVE ? NMAX : 1];
  exact_body<bf16, ALIVE, 1>(a, queue, s64, sd, ALIVE ? alv : nullptr);
}

// every token into the queue (the exact path for all of them)
__global__ void gate_queue_all(int32_t* queue, int T) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i == 0) queue[0] = T;
  if (i < T) queue[GQ_HEAD + i] = i;
}

static size_t gate_mfma_lds_bytes(int dM, int kw) {
  const size_t ring = (size_t)kw * GM_RING * 4096 * (1 + (dM + 31) / 32);
  const size_t scores = (sizeof(double) + sizeof(float)) * GM_TOK * (dM + 1);
  return ring > scores ? ring : scores;
}

static size_t gate_lds_bytes(int dM) {
  return sizeof(double) * (GATE_TB * GATE_KC + GATE_KC * dM + GATE_TB * (dM + 1));
}

// ---------------------------------------------------------------- backward

constexpr int GD_NT = 128;         // gate backward: tokens per block

// dg[t,j] = w (dw - sum_l w_l dw_l) over alive chosen experts; ds row t gets dg at
// column i*M + u_i for every dimension i.  bf16: ds stores hi and lo bf16 parts
// (columns [0, dM) and [dM, 2dM)) so the MFMA product keeps ~16 mantissa bits.

template <typename E>
__global__ void __launch_bounds__(GD_NT)
gate_dg_kernel(const int32_t* idx, const float* w, const float* dw, const uint8_t* alive, float* dg, E* ds,
               int64_t ds_ld, int T, int d, int M, int k, int dM, float* dbg_part) {
  // One thread per token builds its ds row (fp32, in LDS: rows of dM + 1 words); the
  // block then writes its rows (consecutive tokens, one contiguous range) in 16-byte
  // chunks, and adds each column over its rows in row order for the bias gradient.
  extern __shared__ float rowbuf[];
  constexpr int VEC = 16 / sizeof(E);
  const int tl = threadIdx.x;
  const int t0 = blockIdx.x * GD_NT, t = t0 + tl;
  const int nt = min(GD_NT, T - t0);
  const int SR = dM + 1;
  float* row = rowbuf + tl * SR;
  for (int c = 0; c < dM; ++c) row[c] = 0.f;
  if (t < T) {
    float wv[KMAX], dv[KMAX];
    int id[KMAX];
    float s = 0.f;
#pragma unroll
    for (int j = 0; j < KMAX; ++j) {
      wv[j] = 0.f; dv[j] = 0.f; id[j] = 0;
      if (j < k) {
        id[j] = idx[(int64_t)t * k + j];
        const bool live = alive == nullptr || alive[id[j]] != 0;
        wv[j] = live ? w[(int64_t)t * k + j] : 0.f;
        dv[j] = dw[(int64_t)t * k + j];
        s = fmaf(wv[j], dv[j], s);
      }
    }
#pragma unroll
    for (int j = 0; j < KMAX; ++j) {
      if (j < k) {
        const float gj = wv[j] * (dv[j] - s);
        dg[(int64_t)t * k + j] = gj;
        int rem = id[j];
        for (int i = d - 1; i >= 0; --i) { row[i * M + rem % M] += gj; rem /= M; }
      }
    }
  }
  __syncthreads();
  // bf16: hi parts in columns [0, dM), lo parts in [dM, 2 dM), zeros up to ds_ld
  const int cpr = (int)(ds_ld / VEC);
  for (int q = tl; q < nt * cpr; q += GD_NT) {
    const int r = q / cpr, cb = q % cpr;
    const float* src = rowbuf + r * SR;
    alignas(16) E v[VEC];
#pragma unroll
    for (int e = 0; e < VEC; ++e) {
      const int c = cb * VEC + e;
      if constexpr (sizeof(E) == 2) {
        if (c < dM) v[e] = f2bf(src[c]);
        else if (c < 2 * dM) { const float a = src[c - dM]; v[e] = f2bf(a - bf2f(f2bf(a))); }
        else v[e] = 0;
      } else {
        v[e] = c < dM ? src[c] : 0.f;
      }
    }
    *reinterpret_cast<uint4*>(ds + (int64_t)(t0 + r) * ds_ld + cb * VEC) = *reinterpret_cast<const uint4*>(v);
  }
  if (dbg_part) {
    for (int c = tl; c < dM; c += GD_NT) {
      float a = 0.f;
      for (int r = 0; r < nt; ++r) a += rowbuf[r * SR + c];
      dbg_part[(int64_t)blockIdx.x * dM + c] = a;
    }
  }
}

// offsets of the token splits and the GROUP_K tile prefix for the dWg GEMM
__global__ void gate_split_prep(int32_t* offs, int32_t* tprefix, int nsplit, int split, int T) {
  for (int s = threadIdx.x; s <= nsplit; s += blockDim.x) {
    const int o = s * split;
    offs[s] = o < T ? o : T;
    tprefix[s] = s;
  }
}

// dWg[c][n] = sum over splits of the partial products (hi + lo parts for bf16)
template <typename E>
__global__ void gate_reduce_kernel(const float* part, int nsplit, int64_t rows, int dM, int D,
                                   E* dWg) {
  const int64_t q = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (q >= (int64_t)dM * D) return;
  const int c = (int)(q / D), n = (int)(q % D);
  float s = 0.f;
  for (int sp = 0; sp < nsplit; ++sp) {
    const float* P = part + (int64_t)sp * rows * D;
    s += P[(int64_t)c * D + n];
    if constexpr (sizeof(E) == 2) s += P[(int64_t)(dM + c) * D + n];
  }
  dWg[q] = cvt<E>(s);
}

// dbg[c] = sum over the token blocks of their partial column sums, in block order:
// thread i adds a contiguous run of blocks, then a tree over the threads.
template <typename E>
__global__ void __launch_bounds__(256) gate_dbg_kernel(const float* part, int nblk, int dM, E* dbg) {
  const int c = blockIdx.x;
  const int per = (nblk + 255) / 256;
  const int b0 = threadIdx.x * per, b1 = min(nblk, b0 + per);
  float s = 0.f;
  for (int b = b0; b < b1; ++b) s += part[(int64_t)b * dM + c];
  __shared__ float red[256];
  red[threadIdx.x] = s;
  __syncthreads();
  for (int o = 128; o > 0; o >>= 1) {
    if ((int)threadIdx.x < o) red[threadIdx.x] += red[threadIdx.x + o];
    __syncthreads();
  }
  if (threadIdx.x == 0) dbg[c] = cvt<E>(red[0]);
}

}  // namespace dmoe

using namespace dmoe;

extern "C" int dmoe_gate_topk(const dmoe_dims* dims, const void* x, const void* Wg, const void* bg,
                              const uint8_t* alive, int32_t* idx, float* w, float* g, float* scores,
                              void* ws, void* stream) {
  Shape s;
  int rc = check_dims(dims, &s);
  if (rc) return rc;
  if (s.T == 0) return DMOE_OK;
  if (!x || !Wg || !idx || !w) return DMOE_EINVAL;
  if (!aligned16(x) || !aligned16(Wg)) return DMOE_EUNSUPPORTED;
  GateArgs a{x, Wg, bg, alive, idx, w, g, scores, (int)s.T, (int)s.D, s.d, s.M, s.k, (int)s.dM, (int)s.N};
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  const bool alive_first = (s.flags & DMOE_FLAG_ALIVE_TOPK) != 0;
  const bool mfma = s.dtype == DMOE_BF16 && s.dM <= 3 * 32;
  if (alive_first && (!mfma || (s.flags & DMOE_FLAG_GATE_EXACT))) {
    // TopK among the alive experts: exact scores and a ranking of every cell
    if (!ws) return DMOE_EINVAL;
    if (!aligned16(ws)) return DMOE_EUNSUPPORTED;
    int32_t* queue = reinterpret_cast<int32_t*>(reinterpret_cast<unsigned char*>(ws) + workspace_layout(s).gq_off);
    DMOE_LAUNCH(gate_queue_all, dim3((unsigned)((s.T + 255) / 256)), dim3(256), 0, st, queue, (int)s.T);
    const int xgrid = (int)std::min<int64_t>((s.T + GX_TB - 1) / GX_TB, 1024);
    if (s.dtype == DMOE_BF16)
      DMOE_LAUNCH((gate_exact_kernel<bf16, true>), dim3(xgrid), dim3(GX_NT), 0, st, a, queue);
    else
      DMOE_LAUNCH((gate_exact_kernel<float, true>), dim3(xgrid), dim3(GX_NT), 0, st, a, queue);
    return launch_status();
  }
  if (mfma) {
    if (!ws) return DMOE_EINVAL;
    if (!aligned16(ws)) return DMOE_EUNSUPPORTED;
    // error factor of the MFMA scores (see the certificate above gate_topk_mfma)
    const double u = 1.0 / 8388608.0;
    const double g32 = 32 * u / (1 - 32 * u) + (s.D / 32 + 8) * 2.220446049250313e-16;
    const double gD = (double)s.D * u / (1 - (double)s.D * u);
    int32_t* queue = reinterpret_cast<int32_t*>(reinterpret_cast<unsigned char*>(ws) + workspace_layout(s).gq_off);
    GateMfmaArgs ga{a, s.flags, (float)(g32 / (1 - gD) * 1.0001), queue};
    const int KW = gm_kw(s.D);
    const size_t lds = gate_mfma_lds_bytes((int)s.dM, KW);
    const int CB = (int)((s.dM + 31) / 32);
    auto pick = [&](auto AL) {
      constexpr bool A = decltype(AL)::value;
      return KW == 2 ? (CB == 1 ? gate_topk_mfma<1, 2, A> : CB == 2 ? gate_topk_mfma<2, 2, A> : gate_topk_mfma<3, 2, A>)
                     : (CB == 1 ? gate_topk_mfma<1, 1, A> : CB == 2 ? gate_topk_mfma<2, 1, A> : gate_topk_mfma<3, 1, A>);
    };
    auto kern = alive_first ? pick(std::true_type{}) : pick(std::false_type{});
    if (lds > 65536) {
      (void)hipFuncSetAttribute((const void*)kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
      (void)hipGetLastError();
    }
    fill_zero(queue, sizeof(int32_t), st);
    const dim3 grid((unsigned)((s.T + GM_TOK - 1) / GM_TOK));
    DMOE_LAUNCH_NAMED("gate_topk_mfma", kern, grid, dim3(64 * KW), lds, st, ga);
    // exact recomputation of the queued tokens: persistent blocks over the queue
    if (s.flags & DMOE_FLAG_GATE_EXACT) {
      const int xgrid = (int)std::min<int64_t>((s.T + GX_TB - 1) / GX_TB, 1024);
      DMOE_LAUNCH((gate_exact_kernel<bf16, false>), dim3(xgrid), dim3(GX_NT), 0, st, a, queue);
    } else {
      const int xgrid = (int)std::min<int64_t>(s.T, 1024);
      if (alive_first) DMOE_LAUNCH(gate_exact_sparse_kernel<true>, dim3(xgrid), dim3(GX_NT), 0, st, a, queue);
      else DMOE_LAUNCH(gate_exact_sparse_kernel<false>, dim3(xgrid), dim3(GX_NT), 0, st, a, queue);
    }
  } else {
    // fp32, and bf16 with more than 96 gate columns: exact fp64 scores for every token
    const dim3 grid((unsigned)((s.T + GATE_TB - 1) / GATE_TB));
    const size_t lds = gate_lds_bytes((int)s.dM);
    if (s.dtype == DMOE_BF16) DMOE_LAUNCH(gate_topk_kernel<bf16>, grid, dim3(GATE_NT), lds, st, a);
    else DMOE_LAUNCH(gate_topk_kernel<float>, grid, dim3(GATE_NT), lds, st, a);
  }
  return launch_status();
}

template <typename E>
static int gate_bwd_impl(const Shape& s, const void* x, const int32_t* idx, const float* w,
                         const float* dw, const uint8_t* alive, float* dg, void* dWg, void* dbg,
                         void* ws, hipStream_t st) {
  const Workspace L = workspace_layout(s);
  unsigned char* base = reinterpret_cast<unsigned char*>(ws);
  E* ds = reinterpret_cast<E*>(base + L.ds_off);
  float* part = reinterpret_cast<float*>(base + L.part_off);
  int32_t* offs = reinterpret_cast<int32_t*>(base + L.tiles_off);
  int32_t* tpre = offs + (L.gsplit + 1);
  const int T = (int)s.T, D = (int)s.D, dM = (int)s.dM;
  // the bias gradient's per-block column sums use the forward pass's queue region
  // (calls on one stream do not overlap): ceil(T / 128) x dM floats <= 4 T bytes
  const int gblk = (T + GD_NT - 1) / GD_NT;
  float* dbg_part = dbg ? reinterpret_cast<float*>(base + L.gq_off) : nullptr;
  const size_t dg_lds = (size_t)GD_NT * (dM + 1) * sizeof(float);
  if (dg_lds > 65536) {
    (void)hipFuncSetAttribute((const void*)gate_dg_kernel<E>, hipFuncAttributeMaxDynamicSharedMemorySize, (int)dg_lds);
    (void)hipGetLastError();
  }
  DMOE_LAUNCH(gate_dg_kernel<E>, dim3(gblk), dim3(GD_NT), dg_lds, st, idx, w, dw, alive, dg, ds, L.ds_ld, T,
                     s.d, s.M, s.k, dM, dbg_part);
  // dWg partials: one GROUP_K GEMM group per token split, C[split] = ds_split^T x_split
  constexpr int BM = 64, BN = 128, BK = 32, WM = 2, WN = 2;
  const int rows = (int)L.ds_ld;                     // GEMM M (ds columns incl. lo part/padding)
  const int mt = (rows + BM - 1) / BM, nt = (D + BN - 1) / BN;
  DMOE_LAUNCH(gate_split_prep, dim3(1), dim3(256), 0, st, offs, tpre, (int)L.gsplit,
                     (int)L.gsplit_tokens, T);
  GemmArgs<E> p{};
  p.A = ds; p.lda = L.ds_ld;
  p.B = reinterpret_cast<const E*>(x); p.ldb = D;
  p.C = part; p.ldc = D; p.c_gstride = (int64_t)rows * D;
  p.offsets = offs; p.tprefix = tpre; p.tscale = mt * nt; p.groups = (int)L.gsplit;
  p.M = rows; p.N = D; p.K = 0; p.act = s.act;
  const int tiles = (int)L.gsplit * mt * nt;
  auto kern = grouped_gemm<E, GROUP_K, false, EPI_F32, BM, BN, BK, WM, WN>;
  const size_t lds = gemm_lds_bytes<E, BM, BN, BK, WM, WN>();
  int grid = tiles < 2048 ? tiles : 2048;
  p.chunked = grid >= 8;
  DMOE_LAUNCH_NAMED("grouped_gemm<GROUP_K,EPI_F32> (gate dWg per token split)", kern, dim3(grid),
                    dim3(64 * WM * WN), lds, st, p);
  const int64_t outs = (int64_t)dM * D;
  DMOE_LAUNCH(gate_reduce_kernel<E>, dim3((unsigned)((outs + 255) / 256)), dim3(256), 0, st,
                     part, (int)L.gsplit, (int64_t)rows, dM, D, reinterpret_cast<E*>(dWg));
  if (dbg)
    DMOE_LAUNCH(gate_dbg_kernel<E>, dim3(dM), dim3(256), 0, st, dbg_part, gblk, dM, reinterpret_cast<E*>(dbg));
  return launch_status();
}

extern "C" int dmoe_gate_topk_bwd(const dmoe_dims* dims, const void* x, const int32_t* idx,
                                  const float* w, const float* dw, const uint8_t* alive, float* dg,
                                  void* dWg, void* dbg, void* ws, void* stream) {
  Shape s;
  int rc = check_dims(dims, &s);
  if (rc) return rc;
  if (!dWg) return DMOE_EINVAL;
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  if (s.T == 0) {
    // no tokens: zero gradients (a fill kernel, so the call can be graph-captured)
    fill_zero(dWg, (size_t)s.dM * s.D * s.esz, st);
    if (dbg) fill_zero(dbg, (size_t)s.dM * s.esz, st);
    return launch_status();
  }
  if (!x || !idx || !w || !dw || !dg || !ws) return DMOE_EINVAL;
  if (!aligned16(x) || !aligned16(ws)) return DMOE_EUNSUPPORTED;
  if (s.dtype == DMOE_BF16) return gate_bwd_impl<bf16>(s, x, idx, w, dw, alive, dg, dWg, dbg, ws, st);
  return gate_bwd_impl<float>(s, x, idx, w, dw, alive, dg, dWg, dbg, ws, st);
}
