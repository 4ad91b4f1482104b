// Structured gate, exact TopK over the expert grid and Eq. 1 weights
// (Sec. 3.2, Eq. 1, App. C), plus the gate's backward pass.
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

// Insert (v, id) into a list sorted by (v desc, id asc) holding at most cap items.
// Callers insert in increasing id order, so an equal v goes after the items present.
__device__ __forceinline__ void list_insert_f(float* lv, int* li, int& n, int cap, float v, int id) {
  if (n == cap && !(v > lv[cap - 1])) return;
  int p = n < cap ? n : cap - 1;
  while (p > 0 && lv[p - 1] < v) { lv[p] = lv[p - 1]; li[p] = li[p - 1]; --p; }
  lv[p] = v; li[p] = id;
  if (n < cap) ++n;
}

// Insert (v, flat) into the top list ordered by (v desc, flat asc).
__device__ __forceinline__ void list_insert_d(double* tv, int* tf, int& n, int cap, double v, int f) {
  if (n == cap && !(v > tv[cap - 1] || (v == tv[cap - 1] && f < tf[cap - 1]))) return;
  int p = n < cap ? n : cap - 1;
  while (p > 0 && (tv[p - 1] < v || (tv[p - 1] == v && tf[p - 1] > f))) {
    tv[p] = tv[p - 1]; tf[p] = tf[p - 1]; --p;
  }
  tv[p] = v; tf[p] = f;
  if (n < cap) ++n;
}

// One token's selection: per-dimension top-min(k, M) lists, then the cells whose
// rank product is at most k (the only cells that can be among the k best: a cell
// with per-dimension ranks r_i is beaten by the prod(r_i + 1) - 1 cells that take
// an equal or better index in every dimension), ranked by the fp64 total.  When
// the token's scores span more than 2^26 in magnitude a fp64 total of d fp32
// values may round, the dominance argument no longer holds exactly, and the
// token falls back to ranking every cell of the grid.
__device__ void select_token(const double* s64, const uint8_t* alive,
                             int d, int M, int k, float* lv, int* li, double* tv, int* tf,
                             int32_t* idx_out, float* w_out, float* g_out) {
  const int L = k < M ? k : M;
  // decision scores: fp32 rounding of the fp64 gate scores
  auto s32 = [&](int c) { return (float)s64[c]; };
  // magnitude span of the nonzero scores
  float amax = 0.f, amin = 3.4e38f;
  for (int c = 0; c < d * M; ++c) {
    const float a = fabsf(s32(c));
    if (a > 0.f) { amax = fmaxf(amax, a); amin = fminf(amin, a); }
  }
  const bool exact = !(amax > 0.f) || amax <= amin * 67108864.f;   // 2^26
  int nt = 0;
  if (exact) {
    int cnt[DMAX];
    for (int i = 0; i < d; ++i) {
      cnt[i] = 0;
      for (int u = 0; u < M; ++u)
        list_insert_f(lv + i * (KMAX + 1), li + i * (KMAX + 1), cnt[i], L, s32(i * M + u), u);
    }
    int ncand = 1;
    for (int i = 0; i < d; ++i) ncand *= L;
    for (int q = 0; q < ncand; ++q) {
      int rem = q, prod = 1, flat = 0;
      int r[DMAX];
      for (int i = d - 1; i >= 0; --i) { r[i] = rem % L; rem /= L; prod *= r[i] + 1; }
      if (prod > k) continue;
      double tot = 0.0;
      for (int i = 0; i < d; ++i) {
        tot += (double)lv[i * (KMAX + 1) + r[i]];
        flat = flat * M + li[i * (KMAX + 1) + r[i]];
      }
      list_insert_d(tv, tf, nt, k, tot, flat);
    }
  } else {
    int N = 1;
    for (int i = 0; i < d; ++i) N *= M;
    for (int f = 0; f < N; ++f) {
      double tot = 0.0;
      int rem = f, u[DMAX];
      for (int i = d - 1; i >= 0; --i) { u[i] = rem % M; rem /= M; }
      for (int i = 0; i < d; ++i) tot += (double)s32(i * M + u[i]);
      list_insert_d(tv, tf, nt, k, tot, f);
    }
  }
  // Eq. 1 weights from the exact totals of the chosen experts, over the alive ones
  double gx[KMAX];
  double m = -1.0e308;
  bool any = false;
  for (int j = 0; j < k; ++j) {
    int rem = tf[j], u[DMAX];
    for (int i = d - 1; i >= 0; --i) { u[i] = rem % M; rem /= M; }
    double t = 0.0;
    for (int i = 0; i < d; ++i) t += s64[i * M + u[i]];
    gx[j] = t;
    const bool live = alive == nullptr || alive[tf[j]] != 0;
    if (live) { any = true; m = t > m ? t : m; }
  }
  float ex[KMAX];
  float sum = 0.f;
  for (int j = 0; j < k; ++j) {
    const bool live = alive == nullptr || alive[tf[j]] != 0;
    ex[j] = live ? expf((float)(gx[j] - m)) : 0.f;
    sum += ex[j];
  }
  for (int j = 0; j < k; ++j) {
    idx_out[j] = tf[j];
    w_out[j] = any ? ex[j] / sum : 0.f;
    if (g_out) g_out[j] = (float)gx[j];
  }
}

template <typename E>
__global__ void __launch_bounds__(GATE_NT) gate_topk_kernel(GateArgs a) {
  extern __shared__ __align__(16) unsigned char sm[];
  const int dM = a.dM;
  double* xs = reinterpret_cast<double*>(sm);                         // [TB][KC]
  double* wsT = xs + GATE_TB * GATE_KC;                               // [KC][dM]
  double* s64 = wsT + GATE_KC * dM;                                   // [TB][dM]
  float* lv = reinterpret_cast<float*>(s64 + GATE_TB * dM);                 // [TB][DMAX*(KMAX+1)]
  int* li = reinterpret_cast<int*>(lv + GATE_TB * DMAX * (KMAX + 1));       // [TB][DMAX*(KMAX+1)]
  double* tv = reinterpret_cast<double*>(li + GATE_TB * DMAX * (KMAX + 1)); // [TB][KMAX+1]
  int* tf = reinterpret_cast<int*>(tv + GATE_TB * (KMAX + 1));              // [TB][KMAX+1]

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
        s64[tt * dM + c] = v;
      }
    }
  }
  __syncthreads();
  if (a.scores) {
    for (int q = tid; q < GATE_TB * dM; q += GATE_NT) {
      const int t = t0 + q / dM;
      if (t < a.T) a.scores[(int64_t)t * dM + q % dM] = (float)s64[q];
    }
  }
  if (tid < GATE_TB && t0 + tid < a.T) {
    const int t = t0 + tid;
    select_token(s64 + tid * dM, a.alive, a.d, a.M, a.k,
                 lv + tid * DMAX * (KMAX + 1), li + tid * DMAX * (KMAX + 1), tv + tid * (KMAX + 1),
                 tf + tid * (KMAX + 1),
                 a.idx + (int64_t)t * a.k, a.w + (int64_t)t * a.k,
                 a.g ? a.g + (int64_t)t * a.k : nullptr);
  }
}

// ---------------------------------------------------------------- bf16: MFMA scores + certificate
//
// Scores are computed on bf16 MFMA: products of bf16 values are exact in fp32, 64 of
// them are summed per MFMA chunk in fp32, and the chunk sums are added in fp64.  A
// second MFMA over |x|.|w| gives A = sum_k |x_k w_k|, which bounds the accumulation
// error of each score:  |S - exact| <= delta = (gamma_64 + (D/64 + 8) 2^-52) A,
// gamma_n = n u / (1 - n u) with u = 2^-23 (no assumption about the MFMA's internal
// rounding beyond IEEE single precision operations).  Decision scores of the GPU and
// of an exact computation then differ by at most delta + 1 ulp each, a cell total by
// at most d (delta + ulp) =: E.  If the k+1 best cells (k when k = N) are separated
// by gaps larger than 2E, the exact scores give the same TopK in the same order; such
// tokens are certified.  The others are recomputed with exact fp64 accumulation.

constexpr int GM_TOK = 32;        // tokens per block
constexpr int GM_NT = 256;        // 4 waves, each a quarter of the d_model contraction

struct GateMfmaArgs {
  GateArgs a;
  int flags;
  float gam;                       // gamma_64 + (D/64+8) 2^-52, times 1/(1 - gamma_D)
};

// Certified selection of one token from its fp64 scores s64[dM] and error-bound sums
// ab[dM].  Returns false (writes nothing) when the decision is not certified.
__device__ bool select_token_cert(const double* s64, const float* ab, const uint8_t* alive, int d, int M,
                                  int k, int N, float gam, float* lv, int* li, double* tv, int* tf,
                                  int32_t* idx_out, float* w_out, float* g_out) {
  const int K1 = k < N ? k + 1 : k;             // cells whose order must be certified
  const int L = K1 < M ? K1 : M;
  float amax = 0.f, amin = 3.4e38f, dmax = 0.f;
  for (int c = 0; c < d * M; ++c) {
    const float v = fabsf((float)s64[c]);
    if (v > 0.f) { amax = fmaxf(amax, v); amin = fminf(amin, v); }
    dmax = fmaxf(dmax, gam * ab[c]);
  }
  // fp64 totals of d fp32 values are exact when the magnitudes span < 2^25
  if (amax > 0.f && amax > amin * 33554432.f) return false;
  const double E = (double)d * ((double)dmax + (double)amax * 1.1920928955078125e-7);
  int cnt[DMAX];
  for (int i = 0; i < d; ++i) {
    cnt[i] = 0;
    for (int u = 0; u < M; ++u)
      list_insert_f(lv + i * (KMAX + 1), li + i * (KMAX + 1), cnt[i], L, (float)s64[i * M + u], u);
  }
  int ncand = 1;
  for (int i = 0; i < d; ++i) ncand *= L;
  int nt = 0;
  for (int q = 0; q < ncand; ++q) {
    int rem = q, prod = 1, flat = 0;
    int r[DMAX];
    for (int i = d - 1; i >= 0; --i) { r[i] = rem % L; rem /= L; prod *= r[i] + 1; }
    if (prod > K1) continue;
    double tot = 0.0;
    for (int i = 0; i < d; ++i) {
      tot += (double)lv[i * (KMAX + 1) + r[i]];
      flat = flat * M + li[i * (KMAX + 1) + r[i]];
    }
    list_insert_d(tv, tf, nt, K1, tot, flat);
  }
  for (int j = 0; j + 1 < K1; ++j)
    if (!(tv[j] - tv[j + 1] > 2.0 * E)) return false;
  // Eq. 1 weights from the fp64 totals of the chosen experts, over the alive ones
  double gx[KMAX];
  double m = -1.0e308;
  bool any = false;
  for (int j = 0; j < k; ++j) {
    int rem = tf[j], u[DMAX];
    for (int i = d - 1; i >= 0; --i) { u[i] = rem % M; rem /= M; }
    double t = 0.0;
    for (int i = 0; i < d; ++i) t += s64[i * M + u[i]];
    gx[j] = t;
    if (alive == nullptr || alive[tf[j]] != 0) { any = true; m = t > m ? t : m; }
  }
  float ex[KMAX];
  float sum = 0.f;
  for (int j = 0; j < k; ++j) {
    const bool live = alive == nullptr || alive[tf[j]] != 0;
    ex[j] = live ? expf((float)(gx[j] - m)) : 0.f;
    sum += ex[j];
  }
  for (int j = 0; j < k; ++j) {
    idx_out[j] = tf[j];
    w_out[j] = any ? ex[j] / sum : 0.f;
    if (g_out) g_out[j] = (float)gx[j];
  }
  return true;
}

__global__ void __launch_bounds__(GM_NT) gate_topk_mfma(GateMfmaArgs ga) {
  const GateArgs& a = ga.a;
  extern __shared__ __align__(16) unsigned char sm[];
  const int dM = a.dM;
  double* s64 = reinterpret_cast<double*>(sm);                               // [TOK][dM]
  float* ab = reinterpret_cast<float*>(s64 + GM_TOK * dM);                   // [TOK][dM]
  double* part = reinterpret_cast<double*>(ab + GM_TOK * dM);                // [GM_NT] fallback partials
  float* lv = reinterpret_cast<float*>(part + GM_NT);                        // [TOK][DMAX*(KMAX+1)]
  int* li = reinterpret_cast<int*>(lv + GM_TOK * DMAX * (KMAX + 1));
  double* tv = reinterpret_cast<double*>(li + GM_TOK * DMAX * (KMAX + 1));   // [TOK][KMAX+1]
  int* tf = reinterpret_cast<int*>(tv + GM_TOK * (KMAX + 1));
  int* redo = tf + GM_TOK * (KMAX + 1);                                      // [TOK]
  __shared__ int nredo;

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int t0 = blockIdx.x * GM_TOK;
  const bf16* x = reinterpret_cast<const bf16*>(a.x);
  const bf16* W = reinterpret_cast<const bf16*>(a.Wg);
  const bf16* bg = reinterpret_cast<const bf16*>(a.bg);
  if (tid == 0) nredo = 0;
  const int tok = lane & 31;                                   // token of this lane within the block
  const int trow = min(t0 + tok, a.T - 1);
  const int koff = 8 * (lane >> 5);
  const int CB = (dM + 31) / 32;
  const int KQ = a.D / 4;                                      // this wave's share of d_model
  const int kbeg = wave * KQ;                                  // (D is a multiple of 64; KQ of 16)
  const bool exact_all = (ga.flags & DMOE_FLAG_GATE_EXACT) != 0;
  if (!exact_all) {
    for (int cb = 0; cb < CB; ++cb) {
      const int col = min(cb * 32 + (lane & 31), dM - 1);
      const bf16* xr = x + (int64_t)trow * a.D + kbeg + koff;
      const bf16* wr = W + (int64_t)col * a.D + kbeg + koff;
      double acc[16];
      f32x16_t aacc, c;
#pragma unroll
      for (int r = 0; r < 16; ++r) { acc[r] = 0.0; aacc[r] = 0.f; c[r] = 0.f; }
      // chunks of 16 k; every 4 chunks (64 products) the fp32 sums move to fp64.
      // loads run two chunks ahead of the MFMAs.
      const int nch = KQ / 16;
      uint4 xv[2], wv[2];
      xv[0] = *reinterpret_cast<const uint4*>(xr);
      wv[0] = *reinterpret_cast<const uint4*>(wr);
      if (nch > 1) {
        xv[1] = *reinterpret_cast<const uint4*>(xr + 16);
        wv[1] = *reinterpret_cast<const uint4*>(wr + 16);
      }
      for (int q = 0; q < nch; ++q) {
        const uint4 xq = xv[q & 1], wq = wv[q & 1];
        if (q + 2 < nch) {
          xv[q & 1] = *reinterpret_cast<const uint4*>(xr + 16 * (q + 2));
          wv[q & 1] = *reinterpret_cast<const uint4*>(wr + 16 * (q + 2));
        }
        const uint4 xa = make_uint4(xq.x & 0x7fff7fffu, xq.y & 0x7fff7fffu, xq.z & 0x7fff7fffu, xq.w & 0x7fff7fffu);
        const uint4 wa = make_uint4(wq.x & 0x7fff7fffu, wq.y & 0x7fff7fffu, wq.z & 0x7fff7fffu, wq.w & 0x7fff7fffu);
        c = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, wq), __builtin_bit_cast(bf16x8_t, xq),
                                                   c, 0, 0, 0);
        aacc = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8_t, wa),
                                                      __builtin_bit_cast(bf16x8_t, xa), aacc, 0, 0, 0);
        if ((q & 3) == 3 || q + 1 == nch) {
#pragma unroll
          for (int r = 0; r < 16; ++r) { acc[r] += (double)c[r]; c[r] = 0.f; }
        }
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
                s64[tok * dM + cc] = acc[r] + (bg ? (double)bf2f(bg[cc]) : 0.0);
                ab[tok * dM + cc] = aacc[r];
              } else {
                s64[tok * dM + cc] += acc[r];
                ab[tok * dM + cc] += aacc[r];
              }
            }
          }
        }
        __syncthreads();
      }
    }
  }
  __syncthreads();
  // selection: one thread per token
  if (tid < GM_TOK && t0 + tid < a.T) {
    const int t = t0 + tid;
    bool ok = false;
    if (!exact_all)
      ok = select_token_cert(s64 + tid * dM, ab + tid * dM, a.alive, a.d, a.M, a.k, a.N, ga.gam,
                             lv + tid * DMAX * (KMAX + 1), li + tid * DMAX * (KMAX + 1),
                             tv + tid * (KMAX + 1), tf + tid * (KMAX + 1), a.idx + (int64_t)t * a.k,
                             a.w + (int64_t)t * a.k, a.g ? a.g + (int64_t)t * a.k : nullptr);
    if (!ok) redo[atomicAdd(&nredo, 1)] = tid;
  }
  __syncthreads();
  // tokens without a certificate: exact fp64 scores.  Thread tid takes column tid % dM
  // and k-slice tid / dM of S = GM_NT / dM slices; slices are then added in order.
  const int nr = nredo;
  const int S = dM <= GM_NT ? GM_NT / dM : 1;
  const int KS = (a.D / 8 + S - 1) / S * 8;                   // k per slice, multiple of 8
  for (int i = 0; i < nr; ++i) {
    const int tt = redo[i];
    const int t = t0 + tt;
    double sacc = 0.0;
    const int c = tid % dM, sl = tid / dM;
    if (sl < S) {
      const bf16* xr = x + (int64_t)t * a.D;
      const bf16* wr = W + (int64_t)c * a.D;
      const int k1 = min(a.D, (sl + 1) * KS);
      for (int kk = sl * KS; kk < k1; kk += 8) {
        float xf[8], wf[8];
        Vec<bf16>::unpack(*reinterpret_cast<const uint4*>(xr + kk), xf);
        Vec<bf16>::unpack(*reinterpret_cast<const uint4*>(wr + kk), wf);
#pragma unroll
        for (int q = 0; q < 8; ++q) sacc = fma((double)xf[q], (double)wf[q], sacc);
      }
    }
    part[tid] = sacc;
    __syncthreads();
    if (tid < dM) {
      double v = 0.0;
      for (int q = 0; q < S; ++q) v += part[q * dM + tid];
      s64[tt * dM + tid] = v + (bg ? (double)bf2f(bg[tid]) : 0.0);
    }
    __syncthreads();
  }
  if (tid < nr) {
    const int tt = redo[tid];
    const int t = t0 + tt;
    select_token(s64 + tt * dM, a.alive, a.d, a.M, a.k, lv + tt * DMAX * (KMAX + 1), li + tt * DMAX * (KMAX + 1),
                 tv + tt * (KMAX + 1), tf + tt * (KMAX + 1), a.idx + (int64_t)t * a.k, a.w + (int64_t)t * a.k,
                 a.g ? a.g + (int64_t)t * a.k : nullptr);
  }
  if (a.scores) {
    for (int q = tid; q < GM_TOK * dM; q += GM_NT) {
      const int t = t0 + q / dM;
      if (t < a.T) a.scores[(int64_t)t * dM + q % dM] = (float)s64[q];
    }
  }
}

static size_t gate_mfma_lds_bytes(int dM) {
  return (sizeof(double) + sizeof(float)) * GM_TOK * dM + sizeof(double) * GM_NT +
         (sizeof(float) + sizeof(int)) * GM_TOK * DMAX * (KMAX + 1) +
         (sizeof(double) + sizeof(int)) * GM_TOK * (KMAX + 1) + sizeof(int) * GM_TOK;
}

static size_t gate_lds_bytes(int dM) {
  return sizeof(double) * (GATE_TB * GATE_KC + GATE_KC * dM + GATE_TB * dM) +
         (sizeof(float) + sizeof(int)) * GATE_TB * DMAX * (KMAX + 1) +
         (sizeof(double) + sizeof(int)) * GATE_TB * (KMAX + 1);
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
  (void)ws;
  Shape s;
  int rc = check_dims(dims, &s);
  if (rc) return rc;
  if (s.T == 0) return DMOE_OK;
  if (!x || !Wg || !idx || !w) return DMOE_EINVAL;
  if (!aligned16(x) || !aligned16(Wg)) return DMOE_EUNSUPPORTED;
  GateArgs a{x, Wg, bg, alive, idx, w, g, scores, (int)s.T, (int)s.D, s.d, s.M, s.k, (int)s.dM, (int)s.N};
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  if (s.dtype == DMOE_BF16) {
    // error factor of the MFMA scores (see select_token_cert)
    const double u = 1.0 / 8388608.0;
    const double g64 = 64 * u / (1 - 64 * u) + (s.D / 64 + 8) * 2.220446049250313e-16;
    const double gD = (double)s.D * u / (1 - (double)s.D * u);
    GateMfmaArgs ga{a, s.flags, (float)(g64 / (1 - gD) * 1.0001)};
    const size_t lds = gate_mfma_lds_bytes((int)s.dM);
    static bool attr = false;
    if (!attr) {
      (void)hipFuncSetAttribute((const void*)gate_topk_mfma, hipFuncAttributeMaxDynamicSharedMemorySize,
                                (int)gate_mfma_lds_bytes(DM_MAX));
      (void)hipGetLastError();
      attr = true;
    }
    const dim3 grid((unsigned)((s.T + GM_TOK - 1) / GM_TOK));
    hipLaunchKernelGGL(gate_topk_mfma, grid, dim3(GM_NT), lds, st, ga);
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
