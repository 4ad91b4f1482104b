// Structured gate, exact TopK over the expert grid and Eq. 1 weights
// (Sec. 3.2, Eq. 1, App. C), plus the gate's backward pass.
#include <type_traits>

#include "common.hpp"
#include "gemm.hpp"

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
template <bool CERT>
__device__ __forceinline__ bool select_token(const double* s64, const float* ab, const uint8_t* alive, int d, int M, int k,
                             int N, float gam, int32_t* idx_out, float* w_out, float* g_out) {
  constexpr int CAP = KMAX + 1;
  const int K1 = CERT && k < N ? k + 1 : k;
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
  double tv[CAP];
  int tf[CAP];
#pragma unroll
  for (int p = 0; p < CAP; ++p) { tv[p] = -INFINITY; tf[p] = 0x7fffffff; }
  auto insert = [&](double v, int f) {
#pragma unroll
    for (int p = 0; p < CAP; ++p) {
      const bool sw = v > tv[p] || (v == tv[p] && f < tf[p]);
      const double ov = tv[p];
      const int of = tf[p];
      tv[p] = sw ? v : ov; tf[p] = sw ? f : of;
      v = sw ? ov : v; f = sw ? of : f;
    }
  };
  const bool narrow = !(amax > 0.f) || amax <= amin * (CERT ? 33554432.f : 67108864.f);   // 2^25 / 2^26
  if (CERT && !narrow) return false;
  if (narrow) {
    int ncand = 1;
#pragma unroll
    for (int i = 0; i < DMAX; ++i) if (i < d) ncand *= L;
    for (int q = 0; q < ncand; ++q) {
      int rem = q, prod = 1;
      int r[DMAX];
#pragma unroll
      for (int i = DMAX - 1; i >= 0; --i) {
        r[i] = 0;
        if (i < d) { r[i] = rem % L; rem /= L; prod *= r[i] + 1; }
      }
      if (prod > K1) continue;
      double tot = 0.0;
      int flat = 0;
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
        }
      }
      insert(tot, flat);
    }
  } else {
    for (int f = 0; f < N; ++f) {
      double tot = 0.0;
      int rem = f, u[DMAX];
#pragma unroll
      for (int i = DMAX - 1; i >= 0; --i) { u[i] = 0; if (i < d) { u[i] = rem % M; rem /= M; } }
#pragma unroll
      for (int i = 0; i < DMAX; ++i) if (i < d) tot += (double)(float)s64[i * M + u[i]];
      insert(tot, f);
    }
  }
  if constexpr (CERT) {
    const double E = (double)d * ((double)dmax + (double)amax * 1.1920928955078125e-7);
    bool sep = true;
#pragma unroll
    for (int j = 0; j + 1 < CAP; ++j)
      if (j + 1 < K1) sep = sep && (tv[j] - tv[j + 1] > 2.0 * E);
    if (!sep) return false;
  }
  // Eq. 1 weights from the fp64 totals of the chosen experts, over the alive ones
  double gx[KMAX];
  bool live[KMAX];
  double m = -1.0e308;
  bool any = false;
#pragma unroll
  for (int j = 0; j < KMAX; ++j) {
    gx[j] = 0.0; live[j] = false;
    if (j < k) {
      int rem = tf[j], u[DMAX];
#pragma unroll
      for (int i = DMAX - 1; i >= 0; --i) { u[i] = 0; if (i < d) { u[i] = rem % M; rem /= M; } }
      double t = 0.0;
#pragma unroll
      for (int i = 0; i < DMAX; ++i) if (i < d) t += s64[i * M + u[i]];
      gx[j] = t;
      live[j] = alive == nullptr || alive[tf[j]] != 0;
      if (live[j]) { any = true; m = t > m ? t : m; }
    }
  }
  float ex[KMAX];
  float sum = 0.f;
#pragma unroll
  for (int j = 0; j < KMAX; ++j) {
    ex[j] = j < k && live[j] ? expf((float)(gx[j] - m)) : 0.f;
    sum += ex[j];
  }
#pragma unroll
  for (int j = 0; j < KMAX; ++j) {
    if (j < k) {
      idx_out[j] = tf[j];
      w_out[j] = any ? ex[j] / sum : 0.f;
      if (g_out) g_out[j] = (float)gx[j];
    }
  }
  return true;
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

constexpr int GM_TOK = 32;        // tokens per block
constexpr int GM_NT = 256;        // 4 waves, each a quarter of the d_model contraction
constexpr int GX_NT = 256;        // exact recomputation: threads per token

struct GateMfmaArgs {
  GateArgs a;
  int flags;
  float gam;                       // gamma_32 + (D/32+8) 2^-52, times 1/(1 - gamma_D)
  int32_t* queue;                  // [0] count, [GQ_HEAD + i] token ids
};

__global__ void __launch_bounds__(GM_NT) gate_topk_mfma(GateMfmaArgs ga) {
  const GateArgs& a = ga.a;
  extern __shared__ __align__(16) unsigned char sm[];
  const int dM = a.dM;
  // per-token rows are padded to an odd number of 4- or 8-byte words, so that the 32
  // tokens of a half-wave fall on distinct LDS banks
  const int SLD = dM + 1;
  double* s64 = reinterpret_cast<double*>(sm);                               // [TOK][SLD]
  float* ab = reinterpret_cast<float*>(s64 + GM_TOK * SLD);                  // [TOK][SLD]

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int t0 = blockIdx.x * GM_TOK;
  const bool exact_all = (ga.flags & DMOE_FLAG_GATE_EXACT) != 0;
  if (exact_all) {                       // every token goes to the exact path
    if (tid < GM_TOK && t0 + tid < a.T) ga.queue[GQ_HEAD + atomicAdd(ga.queue, 1)] = t0 + tid;
    return;
  }
  const bf16* x = reinterpret_cast<const bf16*>(a.x);
  const bf16* W = reinterpret_cast<const bf16*>(a.Wg);
  const bf16* bg = reinterpret_cast<const bf16*>(a.bg);
  const int tok = lane & 31;                                   // token of this lane within the block
  const int trow = min(t0 + tok, a.T - 1);
  const int half = lane >> 5;
  const int CB = (dM + 31) / 32;
  // d_model is cut in groups of 64; wave w takes groups w, w+4, ...  Within a group,
  // lane half h holds k = 32h .. 32h+31, four 16-byte loads issued back to back (whole
  // 128-byte lines per row), and MFMA chunk j takes its 8 elements 32h+8j .. 32h+8j+7
  // from both x and Wg, so every product x_k w_k appears once (contraction order permuted).
  const int NG = a.D / 64;
  const int ng = NG > wave ? (NG - wave + 3) / 4 : 0;         // groups of this wave
  for (int cb = 0; cb < CB; ++cb) {
    const int col = min(cb * 32 + (lane & 31), dM - 1);
    const bf16* xr = x + (int64_t)trow * a.D + 64 * wave + 32 * half;
    const bf16* wr = W + (int64_t)col * a.D + 64 * wave + 32 * half;
    double acc[16];
    f32x16_t aacc, c;
#pragma unroll
    for (int r = 0; r < 16; ++r) { acc[r] = 0.0; aacc[r] = 0.f; c[r] = 0.f; }
    // every 2 chunks (32 products) the fp32 sums move to fp64; loads run one group ahead
    uint4 xv[2][4], wv[2][4];
    if (ng > 0) {
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) {
        xv[0][jj] = *reinterpret_cast<const uint4*>(xr + 8 * jj);
        wv[0][jj] = *reinterpret_cast<const uint4*>(wr + 8 * jj);
      }
    }
    // one group: MFMAs on load slot SL while the next group loads into the other slot
    auto group = [&](int gi, auto SLc) {
      constexpr int SL = decltype(SLc)::value;
      if (gi + 1 < ng) {
        const int64_t o = (int64_t)256 * (gi + 1);
#pragma unroll
        for (int jj = 0; jj < 4; ++jj) {
          xv[SL ^ 1][jj] = *reinterpret_cast<const uint4*>(xr + o + 8 * jj);
          wv[SL ^ 1][jj] = *reinterpret_cast<const uint4*>(wr + o + 8 * jj);
        }
      }
#pragma unroll
      for (int jj = 0; jj < 4; ++jj) {
        const uint4 xq = xv[SL][jj], wq = wv[SL][jj];
        const uint4 xa = make_uint4(xq.x & 0x7fff7fffu, xq.y & 0x7fff7fffu, xq.z & 0x7fff7fffu, xq.w & 0x7fff7fffu);
        const uint4 wa = make_uint4(wq.x & 0x7fff7fffu, wq.y & 0x7fff7fffu, wq.z & 0x7fff7fffu, wq.w & 0x7fff7fffu);
        c = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, wq), __builtin_bit_cast(bf16x8_t, xq),
                                                   c, 0, 0, 0);
        aacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, wa),
                                                      __builtin_bit_cast(bf16x8_t, xa), aacc, 0, 0, 0);
        if (jj & 1) {
#pragma unroll
          for (int r = 0; r < 16; ++r) { acc[r] += (double)c[r]; c[r] = 0.f; }
        }
      }
    };
    for (int gi = 0; gi < ng; gi += 2) {
      group(gi, std::integral_constant<int, 0>{});
      if (gi + 1 < ng) group(gi + 1, std::integral_constant<int, 1>{});
    }
    // lane holds token (lane % 32) and columns cb*32 + 8(r/4) + 4(lane/32) + r%4; the four
    // waves' partial sums are added in wave order
    for (int w = 0; w < 4; ++w) {
      if (wave == w) {
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int cc = cb * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
          if (cc < dM) {
            if (w == 0) {
              s64[tok * SLD + cc] = acc[r] + (bg ? (double)bf2f(bg[cc]) : 0.0);
              ab[tok * SLD + cc] = aacc[r];
            } else {
              s64[tok * SLD + cc] += acc[r];
              ab[tok * SLD + cc] += aacc[r];
            }
          }
        }
      }
      __syncthreads();
    }
  }
  // selection: one thread per token; tokens without a certificate go to the queue
  if (tid < GM_TOK && t0 + tid < a.T) {
    const int t = t0 + tid;
    const bool ok = select_token<true>(s64 + tid * SLD, ab + tid * SLD, a.alive, a.d, a.M, a.k, a.N, ga.gam,
                                       a.idx + (int64_t)t * a.k, a.w + (int64_t)t * a.k,
                                       a.g ? a.g + (int64_t)t * a.k : nullptr);
    if (!ok) ga.queue[GQ_HEAD + atomicAdd(ga.queue, 1)] = t;
    if (ok && a.scores)
      for (int c = 0; c < dM; ++c) a.scores[(int64_t)t * dM + c] = (float)s64[tid * SLD + c];
  }
}

// Exact path for the queued tokens: fp64 scores S[c] = sum_k x_k W[c][k] + b[c], then the
// same selection as the fp32 layers.  One block per token at a time (persistent over
// the queue); thread (c, slice) sums a contiguous k-slice with four fp64 accumulators
// over interleaved 8-element groups, and the slices are added in order.
__global__ void __launch_bounds__(GX_NT) gate_exact_kernel(GateArgs a, const int32_t* queue) {
  __shared__ double s64[DM_MAX];
  __shared__ double part[GX_NT];
  const int tid = threadIdx.x;
  const int dM = a.dM;
  const int n = queue[0];
  const bf16* x = reinterpret_cast<const bf16*>(a.x);
  const bf16* W = reinterpret_cast<const bf16*>(a.Wg);
  const bf16* bg = reinterpret_cast<const bf16*>(a.bg);
  const int S = GX_NT / dM;                                  // k-slices (dM <= DM_MAX = 128 -> S >= 2)
  const int KS = (a.D / 32 + S - 1) / S * 32;                // k per slice, multiple of 32
  const int c = tid % dM, sl = tid / dM;
  for (int qi = blockIdx.x; qi < n; qi += gridDim.x) {
    const int t = queue[GQ_HEAD + qi];
    double acc4[4] = {0.0, 0.0, 0.0, 0.0};
    if (sl < S) {
      const bf16* xr = x + (int64_t)t * a.D;
      const bf16* wr = W + (int64_t)c * a.D;
      const int k1 = min(a.D, (sl + 1) * KS);
      for (int kk = sl * KS; kk < k1; kk += 32) {
        uint4 xv[4], wv[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          xv[u] = *reinterpret_cast<const uint4*>(xr + kk + 8 * u);
          wv[u] = *reinterpret_cast<const uint4*>(wr + kk + 8 * u);
        }
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          float xf[8], wf[8];
          Vec<bf16>::unpack(xv[u], xf);
          Vec<bf16>::unpack(wv[u], wf);
#pragma unroll
          for (int q = 0; q < 8; ++q) acc4[u] = fma((double)xf[q], (double)wf[q], acc4[u]);
        }
      }
    }
    part[tid] = (acc4[0] + acc4[1]) + (acc4[2] + acc4[3]);
    __syncthreads();
    if (tid < dM) {
      double v = 0.0;
      for (int q = 0; q < S; ++q) v += part[q * dM + tid];
      s64[tid] = v + (bg ? (double)bf2f(bg[tid]) : 0.0);
    }
    __syncthreads();
    if (tid == 0)
      select_token<false>(s64, nullptr, a.alive, a.d, a.M, a.k, a.N, 0.f, a.idx + (int64_t)t * a.k,
                          a.w + (int64_t)t * a.k, a.g ? a.g + (int64_t)t * a.k : nullptr);
    if (a.scores && tid < dM) a.scores[(int64_t)t * dM + tid] = (float)s64[tid];
    __syncthreads();
  }
}

static size_t gate_mfma_lds_bytes(int dM) {
  return (sizeof(double) + sizeof(float)) * GM_TOK * (dM + 1);
}

static size_t gate_lds_bytes(int dM) {
  return sizeof(double) * (GATE_TB * GATE_KC + GATE_KC * dM + GATE_TB * (dM + 1));
}

// ---------------------------------------------------------------- backward

// dg[t,j] = w (dw - sum_l w_l dw_l) over alive chosen experts; ds row t gets dg at
// column i*M + u_i for every dimension i.  bf16: ds stores hi and lo bf16 parts
// (columns [0, dM) and [dM, 2dM)) so the MFMA product keeps ~16 mantissa bits.
template <typename E>
__global__ void gate_dg_kernel(const int32_t* idx, const float* w, const float* dw,
                               const uint8_t* alive, float* dg, E* ds, int64_t ds_ld,
                               int T, int d, int M, int k, int dM) {
  const int t = blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= T) return;
  float wv[KMAX], dv[KMAX];
  int id[KMAX];
  float s = 0.f;
  for (int j = 0; j < k; ++j) {
    id[j] = idx[(int64_t)t * k + j];
    const bool live = alive == nullptr || alive[id[j]] != 0;
    wv[j] = live ? w[(int64_t)t * k + j] : 0.f;
    dv[j] = dw[(int64_t)t * k + j];
    s = fmaf(wv[j], dv[j], s);
  }
  float row[DM_MAX];
  for (int c = 0; c < dM; ++c) row[c] = 0.f;
  for (int j = 0; j < k; ++j) {
    const float gj = wv[j] * (dv[j] - s);
    dg[(int64_t)t * k + j] = gj;
    int rem = id[j];
    for (int i = d - 1; i >= 0; --i) { row[i * M + rem % M] += gj; rem /= M; }
  }
  E* out = ds + (int64_t)t * ds_ld;
  if constexpr (sizeof(E) == 2) {
    for (int c = 0; c < dM; ++c) {
      const bf16 hi = f2bf(row[c]);
      out[c] = hi;
      out[dM + c] = f2bf(row[c] - bf2f(hi));
    }
    for (int c = 2 * dM; c < ds_ld; ++c) out[c] = 0;
  } else {
    for (int c = 0; c < dM; ++c) out[c] = row[c];
    for (int c = dM; c < ds_ld; ++c) out[c] = 0.f;
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

// dbg[c] = sum_t ds[t][c] (fixed order: per-thread strided sums, then a tree)
template <typename E>
__global__ void gate_dbg_kernel(const E* ds, int64_t ds_ld, int T, int dM, E* dbg) {
  const int c = blockIdx.x;
  float s = 0.f;
  for (int t = threadIdx.x; t < T; t += blockDim.x) {
    const E* r = ds + (int64_t)t * ds_ld;
    s += ldf(r + c);
    if constexpr (sizeof(E) == 2) s += ldf(r + dM + c);
  }
  __shared__ float red[256];
  red[threadIdx.x] = s;
  __syncthreads();
  for (int o = blockDim.x / 2; o > 0; o >>= 1) {
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
  if (s.dtype == DMOE_BF16) {
    if (!ws) return DMOE_EINVAL;
    if (!aligned16(ws)) return DMOE_EUNSUPPORTED;
    // error factor of the MFMA scores (see select_token_cert)
    const double u = 1.0 / 8388608.0;
    const double g32 = 32 * u / (1 - 32 * u) + (s.D / 32 + 8) * 2.220446049250313e-16;
    const double gD = (double)s.D * u / (1 - (double)s.D * u);
    int32_t* queue = reinterpret_cast<int32_t*>(reinterpret_cast<unsigned char*>(ws) + workspace_layout(s).gq_off);
    GateMfmaArgs ga{a, s.flags, (float)(g32 / (1 - gD) * 1.0001), queue};
    const size_t lds = gate_mfma_lds_bytes((int)s.dM);
    static bool attr = false;
    if (!attr) {
      (void)hipFuncSetAttribute((const void*)gate_topk_mfma, hipFuncAttributeMaxDynamicSharedMemorySize,
                                (int)gate_mfma_lds_bytes(DM_MAX));
      (void)hipGetLastError();
      attr = true;
    }
    fill_zero(queue, sizeof(int32_t), st);
    const dim3 grid((unsigned)((s.T + GM_TOK - 1) / GM_TOK));
    hipLaunchKernelGGL(gate_topk_mfma, grid, dim3(GM_NT), lds, st, ga);
    // exact recomputation of the queued tokens: persistent blocks over the queue
    const int xgrid = (int)std::min<int64_t>(s.T, 1024);
    hipLaunchKernelGGL(gate_exact_kernel, dim3(xgrid), dim3(GX_NT), 0, st, a, queue);
  } else {
    const dim3 grid((unsigned)((s.T + GATE_TB - 1) / GATE_TB));
    const size_t lds = gate_lds_bytes((int)s.dM);
    hipLaunchKernelGGL(gate_topk_kernel<float>, grid, dim3(GATE_NT), lds, st, a);
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
  hipLaunchKernelGGL(gate_dg_kernel<E>, dim3((T + 127) / 128), dim3(128), 0, st, idx, w, dw, alive,
                     dg, ds, L.ds_ld, T, s.d, s.M, s.k, dM);
  // dWg partials: one GROUP_K GEMM group per token split, C[split] = ds_split^T x_split
  constexpr int BM = 64, BN = 128, BK = 32, WM = 2, WN = 2;
  const int rows = (int)L.ds_ld;                     // GEMM M (ds columns incl. lo part/padding)
  const int mt = (rows + BM - 1) / BM, nt = (D + BN - 1) / BN;
  hipLaunchKernelGGL(gate_split_prep, dim3(1), dim3(256), 0, st, offs, tpre, (int)L.gsplit,
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
  hipLaunchKernelGGL(kern, dim3(grid), dim3(64 * WM * WN), lds, st, p);
  const int64_t outs = (int64_t)dM * D;
  hipLaunchKernelGGL(gate_reduce_kernel<E>, dim3((unsigned)((outs + 255) / 256)), dim3(256), 0, st,
                     part, (int)L.gsplit, (int64_t)rows, dM, D, reinterpret_cast<E*>(dWg));
  if (dbg)
    hipLaunchKernelGGL(gate_dbg_kernel<E>, dim3(dM), dim3(256), 0, st, ds, L.ds_ld, T, dM,
                       reinterpret_cast<E*>(dbg));
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
