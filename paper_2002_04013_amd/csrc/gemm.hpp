// Grouped GEMM for the expert blocks (gfx950 MFMA, LDS double buffer, persistent
// tiles with an XCD-aware schedule).
//
// C[m][n] = sum_k A[m][k] * B[n][k] for every group (expert) e:
//   GROUP_M: the m range is expert e's rows [offsets[e], offsets[e+1]) (tokens);
//            K and N are fixed; A rows are K-contiguous; B is expert e's weight,
//            K-contiguous ([N][K], nn.Linear) or N-contiguous ([K][N]).
//   GROUP_K: the k range is expert e's rows (tokens); M and N are fixed; A and B
//            are both stored row-per-token ([K][M] and [K][N]); C is expert e's
//            weight gradient [M][N].
// The MFMA's first operand takes the B tile (n) and its second the A tile (m),
// so each lane's accumulator holds 4 consecutive n of one m: 8/16-byte stores.
#pragma once

#include "common.hpp"

namespace dmoe {

enum GroupMode { GROUP_M = 0, GROUP_K = 1 };
// EPI_SGD: C holds parameters; C <- C - lr * (A^T B) (the gradient is not stored)
enum Epilogue { EPI_STORE = 0, EPI_BIAS = 1, EPI_BIAS_ACT = 2, EPI_DACT = 3, EPI_F32 = 4, EPI_SGD = 5 };

template <typename E> struct Mma;
template <> struct Mma<bf16> {
  static constexpr int KPL = 8;    // k per lane per operand
  static constexpr int KI = 16;    // k per instruction (v_mfma_f32_32x32x16_bf16)
  __device__ static f32x16_t run(const bf16* a, const bf16* b, f32x16_t c) {
    const bf16x8_t av = *reinterpret_cast<const bf16x8_t*>(a);
    const bf16x8_t bv = *reinterpret_cast<const bf16x8_t*>(b);
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, bv, c, 0, 0, 0);
  }
};
template <> struct Mma<float> {
  static constexpr int KPL = 1;
  static constexpr int KI = 2;     // v_mfma_f32_32x32x2_f32
  __device__ static f32x16_t run(const float* a, const float* b, f32x16_t c) {
    return __builtin_amdgcn_mfma_f32_32x32x2f32(*a, *b, c, 0, 0, 0);
  }
};

template <typename E>
struct GemmArgs {
  const E* A; int64_t lda;
  const E* B; int64_t ldb; int64_t b_gstride;      // GROUP_M: elements between experts' B
  void* C; int64_t ldc; int64_t c_gstride;         // GROUP_K: elements between experts' C
  void* C2;                                        // EPI_BIAS_ACT: activation output
  const E* bias; int64_t bias_gstride;             // EPI_BIAS*: per-expert bias [N]
  const E* aux;                                    // EPI_DACT: pre-activation, layout of C
  const int32_t* offsets;                          // [groups+1]
  const int32_t* tprefix;                          // [groups+1] prefix of tile units
  int tscale;                                      // tiles per unit of tprefix
  int groups;
  int M, N, K;                                     // fixed dims (M unused for GROUP_M, K for GROUP_K)
  int act;
  int chunked;                                     // XCD-chunked schedule (grid >= 8)
  float lr;                                        // EPI_SGD: step size
};

// K-contiguous tile (R rows x BK): element (r, k) at base[r * ld + k].
template <typename E, int R, int BK, int NT>
struct TileKC {
  static constexpr int VEC = 16 / sizeof(E);
  static constexpr int CPR = BK / VEC;
  static constexpr int TOT = R * CPR;
  static constexpr int NCH = (TOT + NT - 1) / NT;
  uint4 v[NCH];
  __device__ __forceinline__ void load(const E* base, int64_t ld, int rvalid, int tid) {
#pragma unroll
    for (int i = 0; i < NCH; ++i) {
      const int q = tid + i * NT;
      const int r = q / CPR, c = q % CPR;
      v[i] = make_uint4(0, 0, 0, 0);
      if ((TOT % NT == 0 || q < TOT) && r < rvalid)
        v[i] = *reinterpret_cast<const uint4*>(base + (int64_t)r * ld + c * VEC);
    }
  }
  __device__ __forceinline__ void store(E* lds, int ldl, int tid) const {
#pragma unroll
    for (int i = 0; i < NCH; ++i) {
      const int q = tid + i * NT;
      const int r = q / CPR, c = q % CPR;
      if (TOT % NT == 0 || q < TOT)
        *reinterpret_cast<uint4*>(lds + r * ldl + c * VEC) = v[i];
    }
  }
};

// Row-per-k tile (R x BK, stored [k][r]): element (r, k) at base[k * ld + r].
// Each thread loads TK rows of k (16 bytes of consecutive r each) and writes the
// transposed block into LDS so that k is contiguous there.
template <typename E, int R, int BK, int NT>
struct TileT {
  static constexpr int VEC = 16 / sizeof(E);
  static constexpr int TK = 4;
  static constexpr int RB = R / VEC;
  static constexpr int KB = BK / TK;
  static constexpr int TOT = RB * KB;
  static constexpr int NB = (TOT + NT - 1) / NT;
  static_assert(R % VEC == 0 && BK % TK == 0, "tile shape");
  uint4 v[NB][TK];
  __device__ __forceinline__ void load(const E* base, int64_t ld, int rvalid, int kvalid, int tid) {
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      const int q = tid + b * NT;
      const int rb = q % RB, kb = q / RB;
#pragma unroll
      for (int t = 0; t < TK; ++t) {
        const int k = kb * TK + t;
        v[b][t] = make_uint4(0, 0, 0, 0);
        if ((TOT % NT == 0 || q < TOT) && k < kvalid && rb * VEC < rvalid)
          v[b][t] = *reinterpret_cast<const uint4*>(base + (int64_t)k * ld + rb * VEC);
      }
    }
  }
  __device__ __forceinline__ void store(E* lds, int ldl, int tid) const {
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      const int q = tid + b * NT;
      if (!(TOT % NT == 0 || q < TOT)) continue;
      const int rb = q % RB, kb = q / RB;
      E* dst = lds + (rb * VEC) * ldl + kb * TK;
      if constexpr (sizeof(E) == 2) {
        // 8 rows of r, 4 k each: row i takes half (i & 1) of word (i >> 1) of every k
#pragma unroll
        for (int i = 0; i < VEC; ++i) {
          uint32_t w[TK];
#pragma unroll
          for (int t = 0; t < TK; ++t) {
            const uint4 u = v[b][t];
            const uint32_t word = (i >> 1) == 0 ? u.x : (i >> 1) == 1 ? u.y : (i >> 1) == 2 ? u.z : u.w;
            w[t] = (i & 1) ? (word >> 16) : (word & 0xffffu);
          }
          *reinterpret_cast<uint2*>(dst + i * ldl) = make_uint2(w[0] | (w[1] << 16), w[2] | (w[3] << 16));
        }
      } else {
#pragma unroll
        for (int i = 0; i < VEC; ++i) {
          uint32_t w[TK];
#pragma unroll
          for (int t = 0; t < TK; ++t) {
            const uint4 u = v[b][t];
            w[t] = i == 0 ? u.x : i == 1 ? u.y : i == 2 ? u.z : u.w;
          }
          *reinterpret_cast<uint4*>(dst + i * ldl) = make_uint4(w[0], w[1], w[2], w[3]);
        }
      }
    }
  }
};

// Tile lookup: expert e owning global tile L; expert e's tiles start at
// tprefix[e] * scale (tprefix is non-decreasing).
__device__ __forceinline__ int find_group(const int32_t* tprefix, int scale, int groups, int L, int lo = 0) {
  int hi = groups;                  // invariant: tprefix[lo]*scale <= L < tprefix[hi]*scale
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (tprefix[mid] * scale <= L) lo = mid; else hi = mid;
  }
  return lo;
}
// Same, for a tile index that is not below the one whose group was `hint`: a block
// walks its tiles in increasing order, so the group is usually `hint` itself (one
// load) or found by searching only above it.
__device__ __forceinline__ int find_group_from(const int32_t* tprefix, int scale, int groups, int L, int hint) {
  if (tprefix[hint + 1] * scale > L) return hint;
  return find_group(tprefix, scale, groups, L, hint + 1);
}

template <typename E, int GM, bool B_KC, int EPI, int BM, int BN, int BK, int WM, int WN>
__global__ void __launch_bounds__(64 * WM * WN)
grouped_gemm(GemmArgs<E> p) {
  constexpr int NT = 64 * WM * WN;
  constexpr int KPL = Mma<E>::KPL, KI = Mma<E>::KI;
  constexpr int PAD = 16 / sizeof(E);
  constexpr int LDL = BK + PAD;
  constexpr int WTM = BM / WM, WTN = BN / WN;        // wave tile
  constexpr int TM = WTM / 32, TN = WTN / 32;        // 32x32 MFMA tiles per wave
  static_assert(TM >= 1 && TN >= 1 && BK % KI == 0, "tile shape");

  extern __shared__ __align__(16) unsigned char smem_raw[];
  E* smem = reinterpret_cast<E*>(smem_raw);
  E* As[2] = {smem, smem + (BM + BN) * LDL};
  E* Bs[2] = {smem + BM * LDL, smem + (BM + BN) * LDL + BM * LDL};

  const int tid = threadIdx.x;
  const int lane = tid & 63, wave = tid >> 6;
  const int wm = wave % WM, wn = wave / WM;
  const int l32 = lane & 31, lhi = lane >> 5;

  const int total = p.tprefix[p.groups] * p.tscale;
  const int nblk = gridDim.x;
  int L, Lend, Lstep;
  if (p.chunked) {
    // Workgroups go to the 8 XCDs round-robin; give each XCD a contiguous share of
    // the tile list so tiles that share a weight slab meet in one L2.
    const int x = blockIdx.x & 7, lb = blockIdx.x >> 3;
    const int per = (nblk - x + 7) >> 3;
    L = (int)(((int64_t)x * total) >> 3) + lb;
    Lend = (int)(((int64_t)(x + 1) * total) >> 3);
    Lstep = per;
  } else {
    L = blockIdx.x; Lend = total; Lstep = nblk;
  }
  const int NTILES = (p.N + BN - 1) / BN;

  for (; L < Lend; L += Lstep) {
    const int e = find_group(p.tprefix, p.tscale, p.groups, L);
    const int q = L - p.tprefix[e] * p.tscale;
    const int off = p.offsets[e];
    const int cnt = p.offsets[e + 1] - off;
    int m0, n0, mvalid, kvalid;
    const E *Ab, *Bb;
    if constexpr (GM == GROUP_M) {
      const int mt_e = (cnt + BM - 1) / BM;
      const int nt = q / mt_e, mt = q % mt_e;
      m0 = mt * BM; n0 = nt * BN;
      mvalid = cnt - m0;
      kvalid = p.K;
      Ab = p.A + (int64_t)(off + m0) * p.lda;
      Bb = p.B + (int64_t)e * p.b_gstride + (B_KC ? (int64_t)n0 * p.ldb : (int64_t)n0);
    } else {
      const int mt = q / NTILES, nt = q % NTILES;
      m0 = mt * BM; n0 = nt * BN;
      mvalid = p.M - m0;
      kvalid = cnt;
      Ab = p.A + (int64_t)off * p.lda + m0;
      Bb = p.B + (int64_t)off * p.ldb + n0;
    }
    const int nvalid = p.N - n0;
    const int nk = (kvalid + BK - 1) / BK;

    f32x16_t acc[TN][TM];
#pragma unroll
    for (int i = 0; i < TN; ++i)
#pragma unroll
      for (int j = 0; j < TM; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

    // operand loaders
    using LA = typename std::conditional<GM == GROUP_M, TileKC<E, BM, BK, NT>, TileT<E, BM, BK, NT>>::type;
    using LB = typename std::conditional<(GM == GROUP_M && B_KC), TileKC<E, BN, BK, NT>, TileT<E, BN, BK, NT>>::type;
    LA la;
    LB lb;
    auto load = [&](int kt) {
      const int k0 = kt * BK;
      if constexpr (GM == GROUP_M) {
        la.load(Ab + k0, p.lda, mvalid, tid);
        if constexpr (B_KC) lb.load(Bb + k0, p.ldb, nvalid, tid);
        else lb.load(Bb + (int64_t)k0 * p.ldb, p.ldb, nvalid, kvalid - k0, tid);
      } else {
        la.load(Ab + (int64_t)k0 * p.lda, p.lda, mvalid, kvalid - k0, tid);
        lb.load(Bb + (int64_t)k0 * p.ldb, p.ldb, nvalid, kvalid - k0, tid);
      }
    };

    if (nk > 0) {
      load(0);
      la.store(As[0], LDL, tid);
      lb.store(Bs[0], LDL, tid);
      __syncthreads();
    }
    for (int kt = 0; kt < nk; ++kt) {
      const int cur = kt & 1;
      if (kt + 1 < nk) load(kt + 1);
      const E* as = As[cur] + (wm * WTM + l32) * LDL + lhi * KPL;
      const E* bs = Bs[cur] + (wn * WTN + l32) * LDL + lhi * KPL;
#pragma unroll
      for (int kk = 0; kk < BK; kk += KI) {
#pragma unroll
        for (int i = 0; i < TN; ++i)
#pragma unroll
          for (int j = 0; j < TM; ++j)
            acc[i][j] = Mma<E>::run(bs + i * 32 * LDL + kk, as + j * 32 * LDL + kk, acc[i][j]);
      }
      if (kt + 1 < nk) {
        la.store(As[cur ^ 1], LDL, tid);
        lb.store(Bs[cur ^ 1], LDL, tid);
      }
      __syncthreads();
    }

    // epilogue: lane holds, for m = m0 + wm*WTM + j*32 + l32, the n values
    //   n0 + wn*WTN + i*32 + 8*g + 4*lhi + {0,1,2,3},  g = 0..3  (acc[i][j][4g..4g+3])
#pragma unroll
    for (int j = 0; j < TM; ++j) {
      const int ml = wm * WTM + j * 32 + l32;
      if (ml >= mvalid) continue;
      int64_t crow;
      if constexpr (GM == GROUP_M) crow = (int64_t)(off + m0 + ml) * p.ldc;
      else crow = (int64_t)e * p.c_gstride + (int64_t)(m0 + ml) * p.ldc;
#pragma unroll
      for (int i = 0; i < TN; ++i) {
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int nl = wn * WTN + i * 32 + 8 * g + 4 * lhi;
          if (nl >= nvalid) continue;
          const int n = n0 + nl;
          float v[4];
#pragma unroll
          for (int r = 0; r < 4; ++r) v[r] = acc[i][j][4 * g + r];
          if constexpr (EPI == EPI_BIAS || EPI == EPI_BIAS_ACT) {
            const E* bp = p.bias + (int64_t)e * p.bias_gstride + n;
#pragma unroll
            for (int r = 0; r < 4; ++r) v[r] += ldf(bp + r);
          }
          if constexpr (EPI == EPI_DACT) {
            const E* hp = p.aux + crow + n;
#pragma unroll
            for (int r = 0; r < 4; ++r) v[r] *= act_bwd(ldf(hp + r), p.act);
          }
          if constexpr (EPI == EPI_SGD) {
            const E* wp = reinterpret_cast<const E*>(p.C) + crow + n;
#pragma unroll
            for (int r = 0; r < 4; ++r) v[r] = ldf(wp + r) - p.lr * v[r];
          }
          if constexpr (EPI == EPI_F32) {
            *reinterpret_cast<float4*>(reinterpret_cast<float*>(p.C) + crow + n) =
                make_float4(v[0], v[1], v[2], v[3]);
          } else {
            E* cp = reinterpret_cast<E*>(p.C) + crow + n;
            if constexpr (sizeof(E) == 2) {
              *reinterpret_cast<uint2*>(cp) =
                  make_uint2((uint32_t)f2bf(v[0]) | ((uint32_t)f2bf(v[1]) << 16),
                             (uint32_t)f2bf(v[2]) | ((uint32_t)f2bf(v[3]) << 16));
            } else {
              *reinterpret_cast<float4*>(cp) = make_float4(v[0], v[1], v[2], v[3]);
            }
            if constexpr (EPI == EPI_BIAS_ACT) {
              float a[4];
#pragma unroll
              for (int r = 0; r < 4; ++r) a[r] = act_fwd(v[r], p.act);
              E* ap = reinterpret_cast<E*>(p.C2) + crow + n;
              if constexpr (sizeof(E) == 2) {
                *reinterpret_cast<uint2*>(ap) =
                    make_uint2((uint32_t)f2bf(a[0]) | ((uint32_t)f2bf(a[1]) << 16),
                               (uint32_t)f2bf(a[2]) | ((uint32_t)f2bf(a[3]) << 16));
              } else {
                *reinterpret_cast<float4*>(ap) = make_float4(a[0], a[1], a[2], a[3]);
              }
            }
          }
        }
      }
    }
  }
}

template <typename E, int BM, int BN, int BK, int WM, int WN>
constexpr size_t gemm_lds_bytes() {
  return (size_t)2 * (BM + BN) * (BK + 16 / sizeof(E)) * sizeof(E);
}

}  // namespace dmoe
