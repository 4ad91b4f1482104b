// The feed-forward block expert of Sec. 4.1 on the per-expert row groups: three
// linear layers with layer normalisation and an activation between them,
//   h1 = x W1^T + b1, a1 = act(LN(h1; g1, be1)), h2 = a1 W2^T + b2,
//   a2 = act(LN(h2; g2, be2)), y = a2 W3^T + b3,
// LN(h; g, b) = g (h - mean) / sqrt(var + eps) + b over the F features of a row
// (biased variance, eps = 1e-5).  The linear layers run on the grouped GEMMs; the
// normalisation, its affine map and the activation are one row kernel, and the
// backward of that step is a row kernel (input gradient) plus a per-expert column
// reduction (scale and shift gradients).
#include "grouped.hpp"

namespace dmoe {

constexpr float LN_EPS = 1e-5f;
constexpr int LN_NT = 256;       // 4 waves; a wave normalises one row at a time
constexpr int LN_CHMAX = 8;      // 16-byte chunks per lane: rows of up to 64*8*VEC values

// Expert that owns row r: the first e with offsets[e + 1] > r.
__device__ __forceinline__ int row_expert(const int32_t* offsets, int N, int r) {
  int lo = 0, hi = N - 1;
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    if (offsets[mid + 1] > r) hi = mid;
    else lo = mid + 1;
  }
  return lo;
}

// fp32 layers use the library's erf; bf16 layers (outputs rounded to 2^-9) the
// erfc-based forms of common.hpp.
// ACT is the activation (DMOE_RELU or DMOE_GELU), fixed at compile time.
template <typename E, int ACT> __device__ __forceinline__ float act_f(float z) {
  if constexpr (sizeof(E) == 4) return act_fwd(z, ACT);
  else return act_fwd_fast(z, ACT);
}
template <typename E, int ACT> __device__ __forceinline__ float act_b(float z) {
  if constexpr (sizeof(E) == 4) return act_bwd(z, ACT);
  else return act_bwd_fast(z, ACT);
}

// Contiguous share of the rows [0, offsets[N]) for wave gw of nw.
struct RowRange { int r0, r1; };
__device__ __forceinline__ RowRange wave_rows(const int32_t* offsets, int N) {
  const int nw = gridDim.x * (LN_NT / 64);
  // the wave index through readfirstlane: every value derived from it is wave-uniform,
  // so row bounds, the row's expert and its statistics come from scalar loads, whose
  // waits do not include the wave's outstanding vector loads and stores
  const int gw = blockIdx.x * (LN_NT / 64) + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int P = offsets[N];
  const int per = (P + nw - 1) / nw;
  const int r0 = min(P, gw * per);
  return {r0, min(P, r0 + per)};
}

// a = act(g (h - mean) rstd + b) per row, stats[r] = (mean, rstd), g and b of the
// row's expert.  Lane l holds chunks l, l + 64, ... of the row (16 bytes each).  The
// next row is loaded before this row's results are stored (vector-memory operations
// retire in order, so a row's loads then never wait for the previous row's stores),
// and the expert's g and b stay in registers until the expert changes.
template <typename E, int CH, int ACT>
__global__ void __launch_bounds__(LN_NT)
ln_act_fwd_kernel(const E* h, const int32_t* offsets, int N, int F, const E* gamma, const E* beta,
                  E* a, float* stats) {
  constexpr int VEC = Vec<E>::N;
  const int lane = threadIdx.x & 63;
  const RowRange rr = wave_rows(offsets, N);
  if (rr.r0 >= rr.r1) return;
  const int nch = F / VEC;
  const float invF = 1.f / (float)F;
  int e = row_expert(offsets, N, rr.r0);
  int eend = offsets[e + 1];
  int eg = -1;                                   // expert whose g, b are in gv, bv
  uint4 hv[CH], gv[CH], bv[CH];
  auto load_row = [&](uint4 (&v)[CH], const E* src) {
#pragma unroll
    for (int i = 0; i < CH; ++i) {
      const int c = lane + 64 * i;
      v[i] = c < nch ? *reinterpret_cast<const uint4*>(src + c * VEC) : make_uint4(0, 0, 0, 0);
    }
  };
  load_row(hv, h + (int64_t)rr.r0 * F);
  for (int r = rr.r0; r < rr.r1; ++r) {
    while (r >= eend) eend = offsets[++e + 1];
    if (e != eg) {
      load_row(gv, gamma + (int64_t)e * F);
      load_row(bv, beta + (int64_t)e * F);
      eg = e;
    }
    uint4 hn[CH];
    if (r + 1 < rr.r1) load_row(hn, h + (int64_t)(r + 1) * F);
    float s = 0.f;
#pragma unroll
    for (int i = 0; i < CH; ++i) {
      float x[VEC];
      Vec<E>::unpack(hv[i], x);
#pragma unroll
      for (int j = 0; j < VEC; ++j) s += x[j];
    }
    const float mean = wave_sum(s) * invF;
    float q = 0.f;
#pragma unroll
    for (int i = 0; i < CH; ++i) {
      if (lane + 64 * i >= nch) continue;
      float x[VEC];
      Vec<E>::unpack(hv[i], x);
#pragma unroll
      for (int j = 0; j < VEC; ++j) q += (x[j] - mean) * (x[j] - mean);
    }
    const float rstd = 1.f / sqrtf(wave_sum(q) * invF + LN_EPS);
    E* ar = a + (int64_t)r * F;
#pragma unroll
    for (int i = 0; i < CH; ++i) {
      const int c = lane + 64 * i;
      if (c >= nch) continue;
      float x[VEC], g[VEC], b[VEC], o[VEC];
      Vec<E>::unpack(hv[i], x);
      Vec<E>::unpack(gv[i], g);
      Vec<E>::unpack(bv[i], b);
#pragma unroll
      for (int j = 0; j < VEC; ++j) o[j] = act_f<E, ACT>(fmaf(g[j], (x[j] - mean) * rstd, b[j]));
      *reinterpret_cast<uint4*>(ar + c * VEC) = Vec<E>::pack(o);
    }
    if (lane == 0) *reinterpret_cast<float2*>(stats + 2 * (int64_t)r) = make_float2(mean, rstd);
    if (r + 1 < rr.r1) {
#pragma unroll
      for (int i = 0; i < CH; ++i) hv[i] = hn[i];
    }
  }
}

// Input gradient of the normalisation step, per row:
//   n = (h - mean) rstd, z = g n + b, dn = da act'(z) g,
//   dh = rstd (dn - mean_f(dn) - n mean_f(dn n)).
// The whole row is read before it is written, so dh may alias da.  dn is kept in fp32
// registers between the two passes (the second pass only recomputes n); g and b are
// read per chunk (the expert's two rows stay in L1), so that several waves share a
// SIMD and one wave's arithmetic covers another's loads.
template <typename E, int CH, int ACT>
__global__ void __launch_bounds__(LN_NT)
ln_act_bwd_rows_kernel(const E* h, const float* stats, const int32_t* offsets, int N, int F, const E* gamma,
                       const E* beta, const E* da, E* dh) {
  constexpr int VEC = Vec<E>::N;
  const int lane = threadIdx.x & 63;
  const RowRange rr = wave_rows(offsets, N);
  if (rr.r0 >= rr.r1) return;
  const int nch = F / VEC;
  const float invF = 1.f / (float)F;
  int e = row_expert(offsets, N, rr.r0);
  int eend = offsets[e + 1];
  for (int r = rr.r0; r < rr.r1; ++r) {
    while (r >= eend) eend = offsets[++e + 1];
    const E* gr = gamma + (int64_t)e * F;
    const E* br = beta + (int64_t)e * F;
    uint4 hv[CH], dv[CH];
#pragma unroll
    for (int i = 0; i < CH; ++i) {
      const int c = lane + 64 * i;
      hv[i] = c < nch ? *reinterpret_cast<const uint4*>(h + (int64_t)r * F + c * VEC) : make_uint4(0, 0, 0, 0);
      dv[i] = c < nch ? *reinterpret_cast<const uint4*>(da + (int64_t)r * F + c * VEC) : make_uint4(0, 0, 0, 0);
    }
    const float2 st = *reinterpret_cast<const float2*>(stats + 2 * (int64_t)r);
    const float mean = st.x, rstd = st.y;
    float dnf[CH][VEC];
    float s1 = 0.f, s2 = 0.f;
#pragma unroll
    for (int i = 0; i < CH; ++i) {
      const int c = lane + 64 * i;
#pragma unroll
      for (int j = 0; j < VEC; ++j) dnf[i][j] = 0.f;
      if (c >= nch) continue;
      const uint4 gq = *reinterpret_cast<const uint4*>(gr + c * VEC);
      const uint4 bq = *reinterpret_cast<const uint4*>(br + c * VEC);
      float x[VEC], d[VEC], g[VEC], b[VEC];
      Vec<E>::unpack(hv[i], x);
      Vec<E>::unpack(dv[i], d);
      Vec<E>::unpack(gq, g);
      Vec<E>::unpack(bq, b);
#pragma unroll
      for (int j = 0; j < VEC; ++j) {
        const float n = (x[j] - mean) * rstd;
        const float dn = d[j] * act_b<E, ACT>(fmaf(g[j], n, b[j])) * g[j];
        dnf[i][j] = dn;
        s1 += dn;
        s2 += dn * n;
      }
    }
    const float m1 = wave_sum(s1) * invF, m2 = wave_sum(s2) * invF;
    E* out = dh + (int64_t)r * F;
#pragma unroll
    for (int i = 0; i < CH; ++i) {
      const int c = lane + 64 * i;
      if (c >= nch) continue;
      float x[VEC], o[VEC];
      Vec<E>::unpack(hv[i], x);
#pragma unroll
      for (int j = 0; j < VEC; ++j) {
        const float n = (x[j] - mean) * rstd;
        o[j] = rstd * (dnf[i][j] - m1 - n * m2);
      }
      *reinterpret_cast<uint4*>(out + c * VEC) = Vec<E>::pack(o);
    }
  }
}

// Scale and shift gradients of the normalisation step, per expert e and feature f:
//   dgamma[e][f] = sum over e's rows of da act'(z) n,  dbeta[e][f] = sum of da act'(z).
// Block (x, e) takes 256 * VEC features of expert e and walks its rows in order.
// Experts without rows are left untouched.
template <typename E, int ACT>
__global__ void __launch_bounds__(256)
ln_act_bwd_params_kernel(const E* h, const float* stats, const int32_t* offsets, int F, const E* gamma,
                         const E* beta, const E* da, E* dgamma, E* dbeta) {
  constexpr int VEC = Vec<E>::N;
  const int e = blockIdx.y;
  const int r0 = offsets[e], r1 = offsets[e + 1];
  if (r1 == r0) return;
  const int c = (blockIdx.x * 256 + threadIdx.x) * VEC;
  if (c >= F) return;
  float g[VEC], b[VEC], ag[VEC], ab[VEC];
  Vec<E>::unpack(*reinterpret_cast<const uint4*>(gamma + (int64_t)e * F + c), g);
  Vec<E>::unpack(*reinterpret_cast<const uint4*>(beta + (int64_t)e * F + c), b);
#pragma unroll
  for (int j = 0; j < VEC; ++j) ag[j] = ab[j] = 0.f;
  constexpr int U = 4;
  int r = r0;
  for (; r + U <= r1; r += U) {
    uint4 hv[U], dv[U];
    float2 st[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      hv[u] = *reinterpret_cast<const uint4*>(h + (int64_t)(r + u) * F + c);
      dv[u] = *reinterpret_cast<const uint4*>(da + (int64_t)(r + u) * F + c);
      st[u] = *reinterpret_cast<const float2*>(stats + 2 * (int64_t)(r + u));
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      float x[VEC], d[VEC];
      Vec<E>::unpack(hv[u], x);
      Vec<E>::unpack(dv[u], d);
#pragma unroll
      for (int j = 0; j < VEC; ++j) {
        const float n = (x[j] - st[u].x) * st[u].y;
        const float dz = d[j] * act_b<E, ACT>(fmaf(g[j], n, b[j]));
        ag[j] += dz * n;
        ab[j] += dz;
      }
    }
  }
  for (; r < r1; ++r) {
    float x[VEC], d[VEC];
    Vec<E>::unpack(*reinterpret_cast<const uint4*>(h + (int64_t)r * F + c), x);
    Vec<E>::unpack(*reinterpret_cast<const uint4*>(da + (int64_t)r * F + c), d);
    const float2 st = *reinterpret_cast<const float2*>(stats + 2 * (int64_t)r);
#pragma unroll
    for (int j = 0; j < VEC; ++j) {
      const float n = (x[j] - st.x) * st.y;
      const float dz = d[j] * act_b<E, ACT>(fmaf(g[j], n, b[j]));
      ag[j] += dz * n;
      ab[j] += dz;
    }
  }
  *reinterpret_cast<uint4*>(dgamma + (int64_t)e * F + c) = Vec<E>::pack(ag);
  *reinterpret_cast<uint4*>(dbeta + (int64_t)e * F + c) = Vec<E>::pack(ab);
}

// chunks per lane for a row of F values: the smallest of 1, 2, 4, 8 that holds it
template <typename E> static int ln_chunks(int64_t F) {
  const int64_t per = (F / Vec<E>::N + 63) / 64;
  return per <= 1 ? 1 : per <= 2 ? 2 : per <= 4 ? 4 : 8;
}
template <typename E> static bool ln_width_ok(int64_t F) {
  return F % Vec<E>::N == 0 && F / Vec<E>::N <= 64 * LN_CHMAX;
}

static int ln_grid(const Shape& s) {
  const int64_t waves = std::max<int64_t>(1, std::min<int64_t>(s.P, 4096));
  return (int)((waves + LN_NT / 64 - 1) / (LN_NT / 64));
}

template <typename E, int ACT>
static void ln_fwd_act(const Shape& s, const int32_t* offsets, const E* h, const E* g, const E* b, E* a,
                       float* stats, hipStream_t st) {
  const int N = (int)s.N, F = (int)s.H, grid = ln_grid(s);
  switch (ln_chunks<E>(F)) {
    case 1: DMOE_LAUNCH((ln_act_fwd_kernel<E, 1, ACT>), dim3(grid), dim3(LN_NT), 0, st, h, offsets, N, F, g, b, a, stats); break;
    case 2: DMOE_LAUNCH((ln_act_fwd_kernel<E, 2, ACT>), dim3(grid), dim3(LN_NT), 0, st, h, offsets, N, F, g, b, a, stats); break;
    case 4: DMOE_LAUNCH((ln_act_fwd_kernel<E, 4, ACT>), dim3(grid), dim3(LN_NT), 0, st, h, offsets, N, F, g, b, a, stats); break;
    default: DMOE_LAUNCH((ln_act_fwd_kernel<E, 8, ACT>), dim3(grid), dim3(LN_NT), 0, st, h, offsets, N, F, g, b, a, stats); break;
  }
}
template <typename E>
static void ln_fwd(const Shape& s, const int32_t* offsets, const E* h, const E* g, const E* b, E* a,
                   float* stats, hipStream_t st) {
  if (s.act == DMOE_RELU) ln_fwd_act<E, DMOE_RELU>(s, offsets, h, g, b, a, stats, st);
  else ln_fwd_act<E, DMOE_GELU>(s, offsets, h, g, b, a, stats, st);
}

// scale and shift gradients first (they read da), then dh (which may overwrite da)
template <typename E, int ACT>
static void ln_bwd_act(const Shape& s, const int32_t* offsets, const E* h, const float* stats, const E* g,
                       const E* b, const E* da, E* dh, E* dg, E* db, hipStream_t st) {
  const int N = (int)s.N, F = (int)s.H, grid = ln_grid(s);
  constexpr int VEC = Vec<E>::N;
  DMOE_LAUNCH((ln_act_bwd_params_kernel<E, ACT>), dim3((unsigned)((F / VEC + 255) / 256), (unsigned)N),
                     dim3(256), 0, st, h, stats, offsets, F, g, b, da, dg, db);
  switch (ln_chunks<E>(F)) {
    case 1: DMOE_LAUNCH((ln_act_bwd_rows_kernel<E, 1, ACT>), dim3(grid), dim3(LN_NT), 0, st, h, stats, offsets, N, F, g, b, da, dh); break;
    case 2: DMOE_LAUNCH((ln_act_bwd_rows_kernel<E, 2, ACT>), dim3(grid), dim3(LN_NT), 0, st, h, stats, offsets, N, F, g, b, da, dh); break;
    case 4: DMOE_LAUNCH((ln_act_bwd_rows_kernel<E, 4, ACT>), dim3(grid), dim3(LN_NT), 0, st, h, stats, offsets, N, F, g, b, da, dh); break;
    default: DMOE_LAUNCH((ln_act_bwd_rows_kernel<E, 8, ACT>), dim3(grid), dim3(LN_NT), 0, st, h, stats, offsets, N, F, g, b, da, dh); break;
  }
}
template <typename E>
static void ln_bwd(const Shape& s, const int32_t* offsets, const E* h, const float* stats, const E* g, const E* b,
                   const E* da, E* dh, E* dg, E* db, hipStream_t st) {
  if (s.act == DMOE_RELU) ln_bwd_act<E, DMOE_RELU>(s, offsets, h, stats, g, b, da, dh, dg, db, st);
  else ln_bwd_act<E, DMOE_GELU>(s, offsets, h, stats, g, b, da, dh, dg, db, st);
}

// ---------------------------------------------------------------- linear layers
// Row-major operands: a layer's weight W [N, n_out, n_in], rows grouped by expert.

// C[rows, n_out] = A[rows, n_in] W_e^T + b_e
template <typename E, typename C>
static void lin_fwd(const Shape& s, const int32_t* offsets, const int32_t* tpre, const E* A, int n_in,
                    const E* W, const E* b, int n_out, E* Cp, hipStream_t st) {
  const int64_t mt_ub = (s.P + C::TMR - 1) / C::TMR + std::min<int64_t>(s.N, s.P);
  const int nt = (n_out + C::BN - 1) / C::BN;
  GemmArgs<E> p = args_m<E>(offsets, tpre, nt, (int)s.N);
  p.A = A; p.lda = n_in;
  p.B = W; p.ldb = n_in; p.b_gstride = (int64_t)n_out * n_in;
  p.C = Cp; p.ldc = n_out;
  p.bias = b; p.bias_gstride = n_out;
  p.N = n_out; p.K = n_in; p.act = s.act;
  if constexpr (sizeof(E) == 2)
    run_gemm2<GROUP_M, false, false, EPI_BIAS, C::BM, C::BN, C::WM, C::WN, C::ST, C::BK, STORE_DIRECT, C::XB>(p, mt_ub * nt, st);
  else
    run_gemm<E, GROUP_M, true, EPI_BIAS, C::BM, C::BN, C::BK, C::WM, C::WN>(p, mt_ub * nt, st);
}

// dA[rows, n_in] = dC[rows, n_out] W_e   (W_e read as (n = input feature, k = output feature))
template <typename E, typename C>
static void lin_dgrad(const Shape& s, const int32_t* offsets, const int32_t* tpre, const E* dC, int n_out,
                      const E* W, int n_in, E* dA, hipStream_t st) {
  const int64_t mt_ub = (s.P + C::TMR - 1) / C::TMR + std::min<int64_t>(s.N, s.P);
  const int nt = (n_in + C::BN - 1) / C::BN;
  GemmArgs<E> p = args_m<E>(offsets, tpre, nt, (int)s.N);
  p.A = dC; p.lda = n_out;
  p.B = W; p.ldb = n_in; p.b_gstride = (int64_t)n_out * n_in;
  p.C = dA; p.ldc = n_in;
  p.N = n_in; p.K = n_out; p.act = s.act;
  if constexpr (sizeof(E) == 2)
    run_gemm2<GROUP_M, false, true, EPI_STORE, C::BM, C::BN, C::WM, C::WN, C::ST, C::BK, STORE_DIRECT, C::XB>(p, mt_ub * nt, st);
  else
    run_gemm<E, GROUP_M, false, EPI_STORE, C::BM, C::BN, C::BK, C::WM, C::WN>(p, mt_ub * nt, st);
}

// dW_e[n_out, n_in] = dC_e^T A_e over the expert's rows
template <typename E, typename CW>
static void lin_wgrad(const Shape& s, const int32_t* offsets, const int32_t* tact, const E* dC, int n_out,
                      const E* A, int n_in, E* dW, hipStream_t st) {
  const int64_t active_ub = std::min<int64_t>(s.N, s.P);
  const int mt = (n_out + CW::BM - 1) / CW::BM, nt = (n_in + CW::BN - 1) / CW::BN;
  GemmArgs<E> p = args_m<E>(offsets, tact, mt * nt, (int)s.N);
  p.A = dC; p.lda = n_out;
  p.B = A; p.ldb = n_in;
  p.C = dW; p.ldc = n_in; p.c_gstride = (int64_t)n_out * n_in;
  p.M = n_out; p.N = n_in; p.act = s.act;
  if constexpr (sizeof(E) == 2)
    run_gemm2<GROUP_K, true, true, EPI_STORE, CW::BM, CW::BN, CW::WM, CW::WN, CW::ST, CW::BK, CW::STO>(p, active_ub * mt * nt, st);
  else
    run_gemm<E, GROUP_K, false, EPI_STORE, CW::BM, CW::BN, CW::BK, CW::WM, CW::WN>(p, active_ub * mt * nt, st);
}

template <typename E>
static void colsum(const Shape& s, const int32_t* offsets, const E* X, int ncols, E* out, hipStream_t st) {
  constexpr int VEC = Vec<E>::N;
  DMOE_LAUNCH((segment_colsum<E>), dim3((unsigned)((ncols / VEC + 255) / 256), (unsigned)s.N), dim3(256), 0,
                     st, X, (int64_t)ncols, offsets, ncols, out, 0.f);
}

template <typename E> struct BlockP {
  const E *W1, *b1, *g1, *be1, *W2, *b2, *g2, *be2, *W3, *b3;
};
template <typename E> struct BlockG {
  E *W1, *b1, *g1, *be1, *W2, *b2, *g2, *be2, *W3, *b3;
};
template <typename E> struct BlockA {
  E *h1, *a1, *h2, *a2;
  float *st1, *st2;
};

template <typename E, typename C>
static void block_fwd(const Shape& s, const int32_t* offsets, const E* xp, const BlockP<E>& q, const BlockA<E>& t,
                      E* yp, int32_t* tpre, hipStream_t st) {
  const int D = (int)s.D, F = (int)s.H;
  DMOE_LAUNCH(tile_plan, dim3(1), dim3(1024), 0, st, offsets, (int)s.N, C::TMR, tpre);
  lin_fwd<E, C>(s, offsets, tpre, xp, D, q.W1, q.b1, F, t.h1, st);
  ln_fwd<E>(s, offsets, t.h1, q.g1, q.be1, t.a1, t.st1, st);
  lin_fwd<E, C>(s, offsets, tpre, t.a1, F, q.W2, q.b2, F, t.h2, st);
  ln_fwd<E>(s, offsets, t.h2, q.g2, q.be2, t.a2, t.st2, st);
  lin_fwd<E, C>(s, offsets, tpre, t.a2, F, q.W3, q.b3, D, yp, st);
}

// g2 holds da2 then dh2, g1 holds da1 then dh1 (each normalisation backward in place).
template <typename E, typename C, typename CW>
static void block_bwd(const Shape& s, const int32_t* offsets, const E* xp, const BlockP<E>& q, const BlockA<E>& t,
                      const E* dyp, E* g1, E* g2, E* dxp, const BlockG<E>& d, int32_t* tpre, hipStream_t st) {
  const int D = (int)s.D, F = (int)s.H;
  const int32_t* tact = tpre + s.N + 1;
  DMOE_LAUNCH(tile_plan, dim3(1), dim3(1024), 0, st, offsets, (int)s.N, C::TMR, tpre);
  lin_wgrad<E, CW>(s, offsets, tact, dyp, D, t.a2, F, d.W3, st);     // dW3 = dy^T a2
  colsum<E>(s, offsets, dyp, D, d.b3, st);                            // db3
  lin_dgrad<E, C>(s, offsets, tpre, dyp, D, q.W3, F, g2, st);        // da2 = dy W3
  ln_bwd<E>(s, offsets, t.h2, t.st2, q.g2, q.be2, g2, g2, d.g2, d.be2, st);
  colsum<E>(s, offsets, g2, F, d.b2, st);                             // db2
  lin_wgrad<E, CW>(s, offsets, tact, g2, F, t.a1, F, d.W2, st);       // dW2 = dh2^T a1
  lin_dgrad<E, C>(s, offsets, tpre, g2, F, q.W2, F, g1, st);         // da1 = dh2 W2
  ln_bwd<E>(s, offsets, t.h1, t.st1, q.g1, q.be1, g1, g1, d.g1, d.be1, st);
  colsum<E>(s, offsets, g1, F, d.b1, st);                             // db1
  lin_wgrad<E, CW>(s, offsets, tact, g1, F, xp, D, d.W1, st);         // dW1 = dh1^T x
  lin_dgrad<E, C>(s, offsets, tpre, g1, F, q.W1, D, dxp, st);        // dx_perm = dh1 W1
}

template <typename E> static BlockP<E> params_of(const dmoe_ffblock_params* p) {
  auto c = [](const void* v) { return reinterpret_cast<const E*>(v); };
  return {c(p->W1), c(p->b1), c(p->g1), c(p->be1), c(p->W2), c(p->b2), c(p->g2), c(p->be2), c(p->W3), c(p->b3)};
}
template <typename E> static BlockG<E> grads_of(const dmoe_ffblock_params* p) {
  auto m = [](void* v) { return reinterpret_cast<E*>(v); };
  return {m(p->W1), m(p->b1), m(p->g1), m(p->be1), m(p->W2), m(p->b2), m(p->g2), m(p->be2), m(p->W3), m(p->b3)};
}
template <typename E> static BlockA<E> acts_of(const dmoe_ffblock_acts* a) {
  auto m = [](void* v) { return reinterpret_cast<E*>(v); };
  return {m(a->h1), m(a->a1), m(a->h2), m(a->a2), a->st1, a->st2};
}

static bool params_ok(const dmoe_ffblock_params* p) {
  if (!p) return false;
  for (const void* v : {p->W1, p->b1, p->g1, p->be1, p->W2, p->b2, p->g2, p->be2, p->W3, p->b3})
    if (!v) return false;
  return true;
}
static bool params_aligned(const dmoe_ffblock_params* p) {
  for (const void* v : {p->W1, p->b1, p->g1, p->be1, p->W2, p->b2, p->g2, p->be2, p->W3, p->b3})
    if (!aligned16(v)) return false;
  return true;
}
static bool acts_ok(const dmoe_ffblock_acts* a) {
  return a && a->h1 && a->a1 && a->st1 && a->h2 && a->a2 && a->st2;
}
static bool acts_aligned(const dmoe_ffblock_acts* a) {
  for (const void* v : {a->h1, a->a1, (void*)a->st1, a->h2, a->a2, (void*)a->st2})
    if (!aligned16(v)) return false;
  return true;
}
static bool ln_width_supported(const Shape& s) {
  return s.dtype == DMOE_BF16 ? ln_width_ok<bf16>(s.H) : ln_width_ok<float>(s.H);
}

}  // namespace dmoe

using namespace dmoe;

extern "C" int dmoe_ln_act_fwd(const dmoe_dims* dims, const int32_t* offsets, const void* h, const void* gamma,
                               const void* beta, void* a, float* stats, void* stream) {
  Shape s;
  int rc = check_dims(dims, &s);
  if (rc) return rc;
  if (s.T == 0) return DMOE_OK;
  if (!offsets || !h || !gamma || !beta || !a || !stats) return DMOE_EINVAL;
  if (!ln_width_supported(s)) return DMOE_EUNSUPPORTED;
  for (const void* q : {h, gamma, beta, (const void*)a, (const void*)stats})
    if (!aligned16(q)) return DMOE_EUNSUPPORTED;
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  if (s.dtype == DMOE_BF16)
    ln_fwd<bf16>(s, offsets, reinterpret_cast<const bf16*>(h), reinterpret_cast<const bf16*>(gamma),
                 reinterpret_cast<const bf16*>(beta), reinterpret_cast<bf16*>(a), stats, st);
  else
    ln_fwd<float>(s, offsets, reinterpret_cast<const float*>(h), reinterpret_cast<const float*>(gamma),
                  reinterpret_cast<const float*>(beta), reinterpret_cast<float*>(a), stats, st);
  return launch_status();
}

extern "C" int dmoe_ln_act_bwd(const dmoe_dims* dims, const int32_t* offsets, const void* h, const float* stats,
                               const void* gamma, const void* beta, const void* da, void* dh, void* dgamma,
                               void* dbeta, void* stream) {
  Shape s;
  int rc = check_dims(dims, &s);
  if (rc) return rc;
  if (s.T == 0) return DMOE_OK;
  if (!offsets || !h || !stats || !gamma || !beta || !da || !dh || !dgamma || !dbeta) return DMOE_EINVAL;
  if (!ln_width_supported(s)) return DMOE_EUNSUPPORTED;
  for (const void* q : {h, (const void*)stats, gamma, beta, da, (const void*)dh, (const void*)dgamma,
                        (const void*)dbeta})
    if (!aligned16(q)) return DMOE_EUNSUPPORTED;
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  if (s.dtype == DMOE_BF16) {
    auto c = [](const void* q) { return reinterpret_cast<const bf16*>(q); };
    auto m = [](void* q) { return reinterpret_cast<bf16*>(q); };
    ln_bwd<bf16>(s, offsets, c(h), stats, c(gamma), c(beta), c(da), m(dh), m(dgamma), m(dbeta), st);
  } else {
    auto c = [](const void* q) { return reinterpret_cast<const float*>(q); };
    auto m = [](void* q) { return reinterpret_cast<float*>(q); };
    ln_bwd<float>(s, offsets, c(h), stats, c(gamma), c(beta), c(da), m(dh), m(dgamma), m(dbeta), st);
  }
  return launch_status();
}

extern "C" int dmoe_expert_ffblock_fwd(const dmoe_dims* dims, const int32_t* offsets, const void* x_perm,
                                       const dmoe_ffblock_params* params, const dmoe_ffblock_acts* acts,
                                       void* y_perm, void* ws, void* stream) {
  Shape s;
  int rc = check_dims(dims, &s);
  if (rc) return rc;
  if (s.T == 0) return DMOE_OK;
  if (!offsets || !x_perm || !params_ok(params) || !acts_ok(acts) || !y_perm || !ws) return DMOE_EINVAL;
  if (!ln_width_supported(s)) return DMOE_EUNSUPPORTED;
  if (!aligned16(x_perm) || !aligned16(y_perm) || !aligned16(ws) || !params_aligned(params) || !acts_aligned(acts))
    return DMOE_EUNSUPPORTED;
  int32_t* tpre = reinterpret_cast<int32_t*>(reinterpret_cast<unsigned char*>(ws) + workspace_layout(s).tiles_off);
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  if (s.dtype == DMOE_BF16) {
    const bf16* xp = reinterpret_cast<const bf16*>(x_perm);
    bf16* yp = reinterpret_cast<bf16*>(y_perm);
    if (use_fat(s)) block_fwd<bf16, G2Fat>(s, offsets, xp, params_of<bf16>(params), acts_of<bf16>(acts), yp, tpre, st);
    else block_fwd<bf16, G2Skinny>(s, offsets, xp, params_of<bf16>(params), acts_of<bf16>(acts), yp, tpre, st);
  } else {
    block_fwd<float, CfgF32>(s, offsets, reinterpret_cast<const float*>(x_perm), params_of<float>(params),
                             acts_of<float>(acts), reinterpret_cast<float*>(y_perm), tpre, st);
  }
  return launch_status();
}

extern "C" int dmoe_expert_ffblock_bwd(const dmoe_dims* dims, const int32_t* offsets, const void* x_perm,
                                       const dmoe_ffblock_params* params, const dmoe_ffblock_acts* acts,
                                       const void* dy_perm, void* g1, void* g2, void* dx_perm,
                                       const dmoe_ffblock_params* grads, void* ws, void* stream) {
  Shape s;
  int rc = check_dims(dims, &s);
  if (rc) return rc;
  if (s.T == 0) return DMOE_OK;
  if (!offsets || !x_perm || !params_ok(params) || !acts_ok(acts) || !dy_perm || !g1 || !g2 || !dx_perm ||
      !params_ok(grads) || !ws)
    return DMOE_EINVAL;
  if (!ln_width_supported(s)) return DMOE_EUNSUPPORTED;
  for (const void* q : {x_perm, dy_perm, (const void*)g1, (const void*)g2, (const void*)dx_perm, (const void*)ws})
    if (!aligned16(q)) return DMOE_EUNSUPPORTED;
  if (!params_aligned(params) || !params_aligned(grads) || !acts_aligned(acts)) return DMOE_EUNSUPPORTED;
  int32_t* tpre = reinterpret_cast<int32_t*>(reinterpret_cast<unsigned char*>(ws) + workspace_layout(s).tiles_off);
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  if (s.dtype == DMOE_BF16) {
    auto c = [](const void* q) { return reinterpret_cast<const bf16*>(q); };
    auto m = [](void* q) { return reinterpret_cast<bf16*>(q); };
    if (use_fat(s))
      block_bwd<bf16, G2Fat, G2DW>(s, offsets, c(x_perm), params_of<bf16>(params), acts_of<bf16>(acts), c(dy_perm),
                                   m(g1), m(g2), m(dx_perm), grads_of<bf16>(grads), tpre, st);
    else
      block_bwd<bf16, G2Skinny, G2DWShort>(s, offsets, c(x_perm), params_of<bf16>(params), acts_of<bf16>(acts),
                                      c(dy_perm), m(g1), m(g2), m(dx_perm), grads_of<bf16>(grads), tpre, st);
  } else {
    auto c = [](const void* q) { return reinterpret_cast<const float*>(q); };
    auto m = [](void* q) { return reinterpret_cast<float*>(q); };
    block_bwd<float, CfgF32, CfgDWF32>(s, offsets, c(x_perm), params_of<float>(params), acts_of<float>(acts),
                                       c(dy_perm), m(g1), m(g2), m(dx_perm), grads_of<float>(grads), tpre, st);
  }
  return launch_status();
}
