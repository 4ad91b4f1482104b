// Dispatch of (token, expert) pairs into per-expert row groups, the weighted
// combine of Eq. 1, and their backward passes.
//
// Dispatch is a stable counting sort by expert, without atomics on row order:
//   1. per block of DISP_CHUNK pairs, an LDS histogram of alive pairs per expert;
//   2. the histograms become each block's starting row per expert relative to the
//      expert's first row (a scan down each column), the counts, and the offsets
//      (an exclusive scan of the counts);
//   3. each block ranks its pairs within every expert in pair order (wave-wide
//      rank from one ballot per bit of the expert id, waves taken in order) and
//      writes pos/row_token;
//   4. each token's row of x is copied to its alive pairs' rows of x_perm.
#include "common.hpp"

namespace dmoe {

constexpr int RT_NT = 256;

template <typename T> struct type_tag { using type = T; };

__global__ void __launch_bounds__(RT_NT)
dispatch_hist(const int32_t* idx, const uint8_t* alive, int P, int N, int32_t* block_hist) {
  extern __shared__ int hist[];
  for (int e = threadIdx.x; e < N; e += RT_NT) hist[e] = 0;
  __syncthreads();
  const int p0 = blockIdx.x * DISP_CHUNK;
  const int p1 = min(P, p0 + DISP_CHUNK);
  for (int p = p0 + threadIdx.x; p < p1; p += RT_NT) {
    const int e = idx[p];
    if (alive == nullptr || alive[e]) atomicAdd(&hist[e], 1);
  }
  __syncthreads();
  int32_t* out = block_hist + (int64_t)blockIdx.x * N;
  for (int e = threadIdx.x; e < N; e += RT_NT) out[e] = hist[e];
}

// 2a. Per expert, the exclusive prefix of its per-block counts over the blocks (in
// place) and its total.  A block takes SCAN_E experts (one per lane, so every access
// is a coalesced row segment) in SCAN_S slices of the block rows; slice sums meet in
// LDS and each slice then rewrites its rows from its own starting value.
constexpr int SCAN_E = 64, SCAN_S = 16;
__global__ void __launch_bounds__(SCAN_E * SCAN_S)
dispatch_scan_cols(int32_t* block_hist, int nb, int N, int32_t* counts) {
  __shared__ int part[SCAN_S][SCAN_E];
  const int el = threadIdx.x % SCAN_E, sl = threadIdx.x / SCAN_E;
  const int e = blockIdx.x * SCAN_E + el;
  const int per = (nb + SCAN_S - 1) / SCAN_S;
  const int b0 = min(nb, sl * per), b1 = min(nb, b0 + per);
  int sum = 0;
  if (e < N)
    for (int b = b0; b < b1; ++b) sum += block_hist[(int64_t)b * N + e];
  part[sl][el] = sum;
  __syncthreads();
  int run = 0;
  for (int q = 0; q < sl; ++q) run += part[q][el];
  if (e < N) {
    for (int b = b0; b < b1; ++b) {
      int32_t* h = block_hist + (int64_t)b * N + e;
      const int c = *h;
      *h = run;
      run += c;
    }
    if (sl == SCAN_S - 1) counts[e] = run;
  }
}

// 2b. offsets = exclusive scan of counts, offsets[N] = total (one block of 1024
// threads; thread q owns experts [q*EPT, (q+1)*EPT)).
__global__ void __launch_bounds__(1024)
dispatch_scan_offsets(const int32_t* counts, int N, int32_t* offsets) {
  __shared__ int sums[1024];
  const int q = threadIdx.x;
  const int EPT = (N + 1023) / 1024;
  const int e0 = min(N, q * EPT), e1 = min(N, e0 + EPT);
  int mine = 0;
  for (int e = e0; e < e1; ++e) mine += counts[e];
  sums[q] = mine;
  __syncthreads();
  for (int o = 1; o < 1024; o <<= 1) {     // inclusive Hillis-Steele scan
    const int v = q >= o ? sums[q - o] : 0;
    __syncthreads();
    sums[q] += v;
    __syncthreads();
  }
  int base = sums[q] - mine;
  for (int e = e0; e < e1; ++e) {
    offsets[e] = base;
    base += counts[e];
  }
  if (q == 1023) offsets[N] = sums[1023];
}

__global__ void __launch_bounds__(RT_NT)
dispatch_scatter(const int32_t* idx, const uint8_t* alive, int P, int N, int k,
                 const int32_t* block_hist, const int32_t* offsets, int32_t* pos, int32_t* row_token) {
  extern __shared__ int base[];
  const int32_t* bh = block_hist + (int64_t)blockIdx.x * N;
  for (int e = threadIdx.x; e < N; e += RT_NT) base[e] = offsets[e] + bh[e];
  __syncthreads();
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int nbits = 32 - __builtin_clz((unsigned)N);              // bits of the largest expert id
  for (int r = 0; r < DISP_CHUNK / RT_NT; ++r) {
    const int p = blockIdx.x * DISP_CHUNK + r * RT_NT + threadIdx.x;
    int e = -1;
    if (p < P) {
      const int e0 = idx[p];
      if (alive == nullptr || alive[e0]) e = e0;
    }
    // lanes of this wave holding the same id (or both none): the intersection, over the
    // id's bits and its sign, of the ballots of lanes that agree with this lane's bit
    uint64_t same = ~0ull;
    for (int b = 0; b < nbits; ++b) {
      const bool bit = (e >> b) & 1;
      const uint64_t on = __ballot(bit);
      same &= bit ? on : ~on;
    }
    {
      const uint64_t neg = __ballot(e < 0);
      same &= e < 0 ? neg : ~neg;
    }
    const int rank = __popcll(same & ((1ull << lane) - 1ull));
    const bool last = ((same >> lane) >> 1) == 0ull;
    int row = -1;
    for (int w = 0; w < RT_NT / 64; ++w) {
      if (wave == w && e >= 0) {
        row = base[e] + rank;
        if (last) base[e] = row + 1;
      }
      __syncthreads();
    }
    if (p < P) {
      pos[p] = row;
      if (row >= 0) row_token[row] = p / k;
    }
  }
}

// 16-byte store with the non-temporal hint, for large outputs written once in whole
// 128-byte lines (a wave store covers 1 KB of one row): such lines are not left in the
// caches as dirty lines that a later kernel's reads must first write back.  Used for
// x_perm, y and dx; dy_perm keeps ordinary stores (the dh GEMM right after it reads it
// faster from the caches: non-temporal measured 5% slower there).  (Partial
// lines written this way lose the caches' write combining.)
__device__ __forceinline__ void store_stream16(void* p, const uint4& v) {
  typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
  __builtin_nontemporal_store(__builtin_bit_cast(u32x4_t, v), reinterpret_cast<u32x4_t*>(p));
}

// x_perm[pos[t,j]] = x[t]: each token's row is read once and written to each of its
// alive pairs' rows (reading per token, not per row, keeps x traffic at one pass).
template <typename E>
__global__ void __launch_bounds__(RT_NT)
gather_rows(const E* x, const int32_t* pos, int T, int k, int D, E* xp) {
  constexpr int VEC = 16 / sizeof(E);
  const int CPR = D / VEC;
  const int64_t total = (int64_t)T * CPR;
  for (int64_t q = (int64_t)blockIdx.x * RT_NT + threadIdx.x; q < total; q += (int64_t)gridDim.x * RT_NT) {
    const int64_t t = q / CPR;
    const int c = (int)(q % CPR);
    const uint4 v = *reinterpret_cast<const uint4*>(x + t * D + c * VEC);
    for (int j = 0; j < k; ++j) {
      const int r = pos[t * k + j];
      if (r >= 0) store_stream16(xp + (int64_t)r * D + c * VEC, v);
    }
  }
}

// y[t] = sum_j w[t,j] y_perm[pos[t,j]]; one wave per token (KM >= k slots held in
// registers, each chunk's row loads issued before they are added in slot order).
template <typename E, int KM>
__global__ void __launch_bounds__(RT_NT)
combine_kernel(const E* yp, const int32_t* pos, const float* w, E* y, int T, int D, int k) {
  constexpr int VEC = 16 / sizeof(E);
  const int t = blockIdx.x * (RT_NT / 64) + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (t >= T) return;
  int pj[KM];
  float wj[KM];
#pragma unroll
  for (int j = 0; j < KM; ++j) {
    pj[j] = j < k ? pos[(int64_t)t * k + j] : -1;
    wj[j] = j < k ? w[(int64_t)t * k + j] : 0.f;
  }
  const int CPR = D / VEC;
  for (int c = lane; c < CPR; c += 64) {
    uint4 rv[KM];
#pragma unroll
    for (int j = 0; j < KM; ++j)
      if (pj[j] >= 0) rv[j] = *reinterpret_cast<const uint4*>(yp + (int64_t)pj[j] * D + c * VEC);
    float acc[VEC];
#pragma unroll
    for (int i = 0; i < VEC; ++i) acc[i] = 0.f;
#pragma unroll
    for (int j = 0; j < KM; ++j) {
      if (pj[j] < 0) continue;
      float v[VEC];
      Vec<E>::unpack(rv[j], v);
#pragma unroll
      for (int i = 0; i < VEC; ++i) acc[i] = fmaf(wj[j], v[i], acc[i]);
    }
    store_stream16(y + (int64_t)t * D + c * VEC, Vec<E>::pack(acc));
  }
}

// dy_perm[pos[t,j]] = w[t,j] dy[t];  dw[t,j] = <dy[t], y_perm[pos[t,j]]>  (as combine:
// KM >= k slots, each chunk's loads issued before use)
template <typename E, int KM>
__global__ void __launch_bounds__(RT_NT)
combine_bwd_kernel(const E* dy, const E* yp, const int32_t* pos, const float* w, E* dyp,
                   float* dw, int T, int D, int k) {
  constexpr int VEC = 16 / sizeof(E);
  const int t = blockIdx.x * (RT_NT / 64) + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (t >= T) return;
  int pj[KM];
  float wj[KM], dot[KM];
#pragma unroll
  for (int j = 0; j < KM; ++j) {
    pj[j] = j < k ? pos[(int64_t)t * k + j] : -1;
    wj[j] = j < k ? w[(int64_t)t * k + j] : 0.f;
    dot[j] = 0.f;
  }
  const int CPR = D / VEC;
  for (int c = lane; c < CPR; c += 64) {
    const uint4 gv = *reinterpret_cast<const uint4*>(dy + (int64_t)t * D + c * VEC);
    uint4 rv[KM];
#pragma unroll
    for (int j = 0; j < KM; ++j)
      if (pj[j] >= 0) rv[j] = *reinterpret_cast<const uint4*>(yp + (int64_t)pj[j] * D + c * VEC);
    float g[VEC];
    Vec<E>::unpack(gv, g);
#pragma unroll
    for (int j = 0; j < KM; ++j) {
      if (pj[j] < 0) continue;
      float v[VEC], o[VEC];
      Vec<E>::unpack(rv[j], v);
      float s = 0.f;
#pragma unroll
      for (int i = 0; i < VEC; ++i) {
        s = fmaf(g[i], v[i], s);
        o[i] = wj[j] * g[i];
      }
      dot[j] += s;
      *reinterpret_cast<uint4*>(dyp + (int64_t)pj[j] * D + c * VEC) = Vec<E>::pack(o);
    }
  }
#pragma unroll
  for (int j = 0; j < KM; ++j) {
    if (j >= k) break;
    const float s = wave_sum(dot[j]);
    if (lane == 0) dw[(int64_t)t * k + j] = pj[j] >= 0 ? s : 0.f;
  }
}


// dx[t] = sum_j dx_perm[pos[t,j]]  (+ sum_j dg[t,j] sum_i Wg[i*M + u_i(idx[t,j])]), one
// wave per token.  The gate share is taken over the token's distinct gate columns c,
// sum_c ds[c] Wg[c] with ds[c] the sum (in term order j, then i from d-1 down) of the dg
// of the chosen experts whose uid digit selects c: the top cells of a grid share digits,
// so there are usually about half as many Wg rows to read as terms.  Lane q < d k holds
// term q; the first lane of each column sums that column's weights; up to GCR columns are
// then kept in registers for the whole row (KM >= k rows and GC columns; any further
// columns are read in a loop).  Each 16-byte chunk issues all its loads before adding:
// rows in slot order, then columns in order of first occurrence.
template <typename E, int KM, int GCR>
__global__ void __launch_bounds__(RT_NT)
dispatch_bwd_kernel(const E* dxp, const int32_t* pos, const int32_t* idx, const float* dg,
                    const E* Wg, E* dx, int T, int D, int k, int d, int M) {
  constexpr int VEC = 16 / sizeof(E);
  const int t = blockIdx.x * (RT_NT / 64) + (threadIdx.x >> 6);
  const int lane = threadIdx.x & 63;
  if (t >= T) return;
  int pj[KM];
#pragma unroll
  for (int j = 0; j < KM; ++j) pj[j] = j < k ? pos[(int64_t)t * k + j] : -1;
  // gate columns: term q = j d + (d - 1 - i) on lane q
  const int nterm = dg != nullptr ? k * d : 0;
  int mycol = -1;
  float myw = 0.f;
  if (lane < nterm) {
    const int j = lane / d, i = d - 1 - lane % d;
    int u = idx[(int64_t)t * k + j];
    for (int r = 0; r < d - 1 - i; ++r) u /= M;
    mycol = i * M + u % M;
    myw = dg[(int64_t)t * k + j];
  }
  float wsum = 0.f;
  bool first = lane < nterm;
  for (int q = 0; q < nterm; ++q) {
    const int cq = __shfl(mycol, q, 64);
    const float wq = __shfl(myw, q, 64);
    if (lane < nterm && cq == mycol) {
      if (q < lane) first = false;
      wsum += wq;
    }
  }
  uint64_t fm = __ballot(first);
  const int ncol = __popcll(fm);
  // every distinct column also in this wave's LDS list (read by the loop over the
  // columns past the register cache, which runs in lanes that may have left the chunk
  // loop's active set, so it cannot take them from other lanes)
  __shared__ int s_col[RT_NT / 64][KMAX * DMAX];
  __shared__ float s_w[RT_NT / 64][KMAX * DMAX];
  const int wv = threadIdx.x >> 6;
  if (first) {
    const int slot = __popcll(fm & ((1ull << lane) - 1ull));
    s_col[wv][slot] = mycol;
    s_w[wv][slot] = wsum;
  }
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  int gcol[GCR];
  float gw[GCR];
#pragma unroll
  for (int g = 0; g < GCR; ++g) {
    const int src = fm ? __builtin_ctzll(fm) : 0;
    gcol[g] = g < ncol ? __shfl(mycol, src, 64) : 0;
    gw[g] = g < ncol ? __shfl(wsum, src, 64) : 0.f;
    fm &= fm ? fm - 1 : 0ull;
  }
  const int CPR = D / VEC;
  for (int c = lane; c < CPR; c += 64) {
    uint4 rv[KM], gv[GCR];
#pragma unroll
    for (int j = 0; j < KM; ++j)
      if (pj[j] >= 0) rv[j] = *reinterpret_cast<const uint4*>(dxp + (int64_t)pj[j] * D + c * VEC);
#pragma unroll
    for (int g = 0; g < GCR; ++g)
      if (g < ncol) gv[g] = *reinterpret_cast<const uint4*>(Wg + (int64_t)gcol[g] * D + c * VEC);
    float acc[VEC];
#pragma unroll
    for (int i = 0; i < VEC; ++i) acc[i] = 0.f;
#pragma unroll
    for (int j = 0; j < KM; ++j) {
      if (pj[j] < 0) continue;
      float v[VEC];
      Vec<E>::unpack(rv[j], v);
#pragma unroll
      for (int i = 0; i < VEC; ++i) acc[i] += v[i];
    }
#pragma unroll
    for (int g = 0; g < GCR; ++g) {
      if (g >= ncol) continue;
      float v[VEC];
      Vec<E>::unpack(gv[g], v);
#pragma unroll
      for (int q = 0; q < VEC; ++q) acc[q] = fmaf(gw[g], v[q], acc[q]);
    }
    for (int g = GCR; g < ncol; ++g) {               // rare: more than GCR distinct columns
      const int col = s_col[wv][g];
      const float w = s_w[wv][g];
      float v[VEC];
      Vec<E>::unpack(*reinterpret_cast<const uint4*>(Wg + (int64_t)col * D + c * VEC), v);
#pragma unroll
      for (int q = 0; q < VEC; ++q) acc[q] = fmaf(w, v[q], acc[q]);
    }
    store_stream16(dx + (int64_t)t * D + c * VEC, Vec<E>::pack(acc));
  }
}

}  // namespace dmoe

using namespace dmoe;

extern "C" int dmoe_dispatch(const dmoe_dims* dims, const void* x, const int32_t* idx,
                             const uint8_t* alive, int32_t* counts, int32_t* offsets,
                             int32_t* row_token, int32_t* pos, void* x_perm, void* ws,
                             void* stream) {
  Shape s;
  int rc = check_dims(dims, &s);
  if (rc) return rc;
  if (!counts || !offsets || !ws || (s.T > 0 && (!x || !idx || !row_token || !pos || !x_perm)))
    return DMOE_EINVAL;
  if (!aligned16(ws) || (s.T > 0 && (!aligned16(x) || !aligned16(x_perm)))) return DMOE_EUNSUPPORTED;
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  const Workspace L = workspace_layout(s);
  int32_t* bh = reinterpret_cast<int32_t*>(reinterpret_cast<unsigned char*>(ws) + L.hist_off);
  const int N = (int)s.N, P = (int)s.P;
  const int nb = (int)L.disp_blocks;
  if (nb > 0)
    DMOE_LAUNCH(dispatch_hist, dim3(nb), dim3(RT_NT), N * sizeof(int), st, idx, alive, P, N, bh);
  DMOE_LAUNCH(dispatch_scan_cols, dim3((N + SCAN_E - 1) / SCAN_E), dim3(SCAN_E * SCAN_S), 0, st, bh, nb,
                     N, counts);
  DMOE_LAUNCH(dispatch_scan_offsets, dim3(1), dim3(1024), 0, st, counts, N, offsets);
  if (nb == 0) return launch_status();
  DMOE_LAUNCH(dispatch_scatter, dim3(nb), dim3(RT_NT), N * sizeof(int), st, idx, alive, P, N,
                     s.k, bh, offsets, pos, row_token);
  const int64_t chunks = s.T * (s.D * (int64_t)s.esz / 16);
  const int grid = (int)std::min<int64_t>((chunks + RT_NT - 1) / RT_NT, 256 * 16);
  if (s.dtype == DMOE_BF16)
    DMOE_LAUNCH(gather_rows<bf16>, dim3(grid), dim3(RT_NT), 0, st, reinterpret_cast<const bf16*>(x),
                       pos, (int)s.T, s.k, (int)s.D, reinterpret_cast<bf16*>(x_perm));
  else
    DMOE_LAUNCH(gather_rows<float>, dim3(grid), dim3(RT_NT), 0, st, reinterpret_cast<const float*>(x),
                       pos, (int)s.T, s.k, (int)s.D, reinterpret_cast<float*>(x_perm));
  return launch_status();
}

extern "C" int dmoe_combine(const dmoe_dims* dims, const void* y_perm, const int32_t* pos,
                            const float* w, void* y, void* stream) {
  Shape s;
  int rc = check_dims(dims, &s);
  if (rc) return rc;
  if (s.T == 0) return DMOE_OK;
  if (!y_perm || !pos || !w || !y) return DMOE_EINVAL;
  if (!aligned16(y_perm) || !aligned16(y)) return DMOE_EUNSUPPORTED;
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  const dim3 grid((unsigned)((s.T + 3) / 4));
  auto go = [&](auto EK, auto KMc) {
    using E = typename decltype(EK)::type;
    constexpr int KM = decltype(KMc)::value;
    const char* kname = std::is_same<E, bf16>::value ? "combine_kernel<bf16>" : "combine_kernel<float>";
    DMOE_LAUNCH_NAMED(kname,
                      (combine_kernel<E, KM>), grid, dim3(RT_NT), 0, st, reinterpret_cast<const E*>(y_perm), pos,
                      w, reinterpret_cast<E*>(y), (int)s.T, (int)s.D, s.k);
  };
  using K4 = std::integral_constant<int, 4>;
  using K8 = std::integral_constant<int, KMAX>;
  if (s.dtype == DMOE_BF16) {
    if (s.k <= 4) go(type_tag<bf16>{}, K4{});
    else go(type_tag<bf16>{}, K8{});
  } else {
    if (s.k <= 4) go(type_tag<float>{}, K4{});
    else go(type_tag<float>{}, K8{});
  }
  return launch_status();
}

extern "C" int dmoe_combine_bwd(const dmoe_dims* dims, const void* dy, const void* y_perm,
                                const int32_t* pos, const float* w, void* dy_perm, float* dw,
                                void* stream) {
  Shape s;
  int rc = check_dims(dims, &s);
  if (rc) return rc;
  if (s.T == 0) return DMOE_OK;
  if (!dy || !y_perm || !pos || !w || !dy_perm || !dw) return DMOE_EINVAL;
  if (!aligned16(dy) || !aligned16(y_perm) || !aligned16(dy_perm)) return DMOE_EUNSUPPORTED;
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  const dim3 grid((unsigned)((s.T + 3) / 4));
  auto go = [&](auto EK, auto KMc) {
    using E = typename decltype(EK)::type;
    constexpr int KM = decltype(KMc)::value;
    const char* kname = std::is_same<E, bf16>::value ? "combine_bwd_kernel<bf16>" : "combine_bwd_kernel<float>";
    DMOE_LAUNCH_NAMED(kname,
                      (combine_bwd_kernel<E, KM>), grid, dim3(RT_NT), 0, st, reinterpret_cast<const E*>(dy),
                      reinterpret_cast<const E*>(y_perm), pos, w, reinterpret_cast<E*>(dy_perm), dw, (int)s.T,
                      (int)s.D, s.k);
  };
  using K4 = std::integral_constant<int, 4>;
  using K8 = std::integral_constant<int, KMAX>;
  if (s.dtype == DMOE_BF16) {
    if (s.k <= 4) go(type_tag<bf16>{}, K4{});
    else go(type_tag<bf16>{}, K8{});
  } else {
    if (s.k <= 4) go(type_tag<float>{}, K4{});
    else go(type_tag<float>{}, K8{});
  }
  return launch_status();
}

extern "C" int dmoe_dispatch_bwd(const dmoe_dims* dims, const void* dx_perm, const int32_t* pos,
                                 const int32_t* idx, const float* dg, const void* Wg, void* dx,
                                 void* stream) {
  Shape s;
  int rc = check_dims(dims, &s);
  if (rc) return rc;
  if (s.T == 0) return DMOE_OK;
  if (!dx_perm || !pos || !dx) return DMOE_EINVAL;
  const bool gate = idx && dg && Wg;
  if (!aligned16(dx_perm) || !aligned16(dx) || (gate && !aligned16(Wg))) return DMOE_EUNSUPPORTED;
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  const dim3 grid((unsigned)((s.T + 3) / 4));
  auto go = [&](auto EK, auto KMc) {
    using E = typename decltype(EK)::type;
    constexpr int KM = decltype(KMc)::value;
    const char* kname = std::is_same<E, bf16>::value ? "dispatch_bwd_kernel<bf16>" : "dispatch_bwd_kernel<float>";
    DMOE_LAUNCH_NAMED(kname,
                      (dispatch_bwd_kernel<E, KM, 8>), grid, dim3(RT_NT), 0, st,
                reinterpret_cast<const E*>(dx_perm), pos, gate ? idx : nullptr, gate ? dg : nullptr,
                reinterpret_cast<const E*>(Wg), reinterpret_cast<E*>(dx), (int)s.T, (int)s.D, s.k, s.d, s.M);
  };
  using K4 = std::integral_constant<int, 4>;
  using K8 = std::integral_constant<int, KMAX>;
  if (s.dtype == DMOE_BF16) {
    if (s.k <= 4) go(type_tag<bf16>{}, K4{});
    else go(type_tag<bf16>{}, K8{});
  } else {
    if (s.k <= 4) go(type_tag<float>{}, K4{});
    else go(type_tag<float>{}, K8{});
  }
  return launch_status();
}
