// Launch helpers shared by the expert blocks: the device-side tile plan of a grouped
// GEMM, per-expert column sums, and the tile shapes and launches of the two grouped
// GEMM implementations (gemm.hpp: fp32; gemm2.hpp: bf16 on gfx950).
#pragma once
#include <algorithm>
#include <atomic>
#include <cstdio>

#include "common.hpp"
#include "gemm.hpp"
#include "gemm2.hpp"

namespace dmoe {

// Tile plan of one FFN call, from the expert row offsets:
//   plan[e]         = sum over experts before e of ceil(rows / BM)   (GROUP_M m-tiles)
//   plan[N + 1 + e] = number of experts before e that have rows      (GROUP_K experts)
// A GEMM with NT n-tiles (GROUP_M) or MT*NT tiles per expert (GROUP_K) scales these.
static __global__ void __launch_bounds__(1024)
tile_plan(const int32_t* offsets, int N, int BM, int32_t* plan) {
  __shared__ int s_mt[1024], s_ac[1024];
  const int q = threadIdx.x;
  const int EPT = (N + 1023) / 1024;
  const int e0 = min(N, q * EPT), e1 = min(N, e0 + EPT);
  int mt = 0, ac = 0;
  for (int e = e0; e < e1; ++e) {
    const int c = offsets[e + 1] - offsets[e];
    mt += (c + BM - 1) / BM;
    ac += c > 0;
  }
  s_mt[q] = mt;
  s_ac[q] = ac;
  __syncthreads();
  for (int o = 1; o < 1024; o <<= 1) {
    const int a = q >= o ? s_mt[q - o] : 0, b = q >= o ? s_ac[q - o] : 0;
    __syncthreads();
    s_mt[q] += a;
    s_ac[q] += b;
    __syncthreads();
  }
  int bm = s_mt[q] - mt, ba = s_ac[q] - ac;
  int32_t* act = plan + N + 1;
  for (int e = e0; e < e1; ++e) {
    plan[e] = bm;
    act[e] = ba;
    const int c = offsets[e + 1] - offsets[e];
    bm += (c + BM - 1) / BM;
    ba += c > 0;
  }
  if (q == 1023) {
    plan[N] = s_mt[1023];
    act[N] = s_ac[1023];
  }
}

// out[e][c] = sum of rows [offsets[e], offsets[e+1]) of column c (experts without rows
// are left untouched); SGD: out[e][c] -= lr * that sum (out holds the parameters).
template <typename E, bool SGD = false>
__global__ void __launch_bounds__(256)
segment_colsum(const E* X, int64_t ld, const int32_t* offsets, int ncols, E* out, float lr = 0.f) {
  constexpr int VEC = 16 / sizeof(E);
  const int e = blockIdx.y;
  const int r0 = offsets[e], r1 = offsets[e + 1];
  if (r1 == r0) return;
  const int c = (blockIdx.x * 256 + threadIdx.x) * VEC;
  if (c >= ncols) return;
  float acc[VEC];
#pragma unroll
  for (int i = 0; i < VEC; ++i) acc[i] = 0.f;
  // rows in order; four loads in flight at a time
  constexpr int U = 4;
  int r = r0;
  for (; r + U <= r1; r += U) {
    uint4 q[U];
#pragma unroll
    for (int u = 0; u < U; ++u) q[u] = *reinterpret_cast<const uint4*>(X + (int64_t)(r + u) * ld + c);
#pragma unroll
    for (int u = 0; u < U; ++u) {
      float v[VEC];
      Vec<E>::unpack(q[u], v);
#pragma unroll
      for (int i = 0; i < VEC; ++i) acc[i] += v[i];
    }
  }
  for (; r < r1; ++r) {
    float v[VEC];
    Vec<E>::unpack(*reinterpret_cast<const uint4*>(X + (int64_t)r * ld + c), v);
#pragma unroll
    for (int i = 0; i < VEC; ++i) acc[i] += v[i];
  }
  uint4* op = reinterpret_cast<uint4*>(out + (int64_t)e * ncols + c);
  if constexpr (SGD) {
    float w[VEC];
    Vec<E>::unpack(*op, w);
#pragma unroll
    for (int i = 0; i < VEC; ++i) acc[i] = w[i] - lr * acc[i];
  }
  *op = Vec<E>::pack(acc);
}

constexpr int MAX_DEVICES = 64;

// The current device, or -1 when it cannot be told or is beyond MAX_DEVICES.
static int current_device() {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= MAX_DEVICES) return -1;
  return dev;
}

// Process state of the library: per device, the compute-unit count and each GEMM
// kernel's resident blocks per compute unit, queried on first use.  Slots are atomics
// (0 = not yet known); threads that race on a first query store the same value.
static int device_cus() {
  static std::atomic<int> cus[MAX_DEVICES];
  const int dev = current_device();
  if (dev < 0) return 256;
  int c = cus[dev].load(std::memory_order_relaxed);
  if (!c) {
    int v = 0;
    if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) v = 0;
    c = v > 0 ? v : 256;
    cus[dev].store(c, std::memory_order_relaxed);
  }
  return c;
}

// Resident blocks per compute unit of kernel `kern` with `nt` threads and `lds` bytes
// of dynamic LDS, cached in `slot` (one per kernel instantiation and device); opts the
// kernel into dynamic LDS beyond 64 KiB first.
static int blocks_per_cu(std::atomic<int>* slots, const void* kern, int nt, size_t lds) {
  const int dev = current_device();
  int nb = dev >= 0 ? slots[dev].load(std::memory_order_relaxed) : 0;
  if (!nb) {
    if (lds > 65536) (void)hipFuncSetAttribute(kern, hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&nb, kern, nt, lds) != hipSuccess || nb < 1) nb = 1;
    (void)hipGetLastError();
    if (dev >= 0) slots[dev].store(nb, std::memory_order_relaxed);
  }
  return nb;
}

template <typename E, int GM, bool B_KC, int EPI, int BM, int BN, int BK, int WM, int WN>
static void run_gemm(GemmArgs<E> p, int64_t tiles_ub, hipStream_t st) {
  if (tiles_ub <= 0) return;
  auto kern = grouped_gemm<E, GM, B_KC, EPI, BM, BN, BK, WM, WN>;
  constexpr int NT = 64 * WM * WN;
  const size_t lds = gemm_lds_bytes<E, BM, BN, BK, WM, WN>();
  static std::atomic<int> per_cu[MAX_DEVICES];
  static const char* name = [] {
    static char b[96];
    snprintf(b, sizeof b, "grouped_gemm<GM=%d,EPI=%d,%dx%d>", GM, EPI, BM, BN);
    return b;
  }();
  const int nb = blocks_per_cu(per_cu, (const void*)kern, NT, lds);
  const int64_t resident = (int64_t)nb * device_cus();
  const int grid = (int)std::min<int64_t>(tiles_ub, resident);
  p.chunked = grid >= 8;
  DMOE_LAUNCH_NAMED(name, kern, dim3(grid), dim3(NT), lds, st, p);
}

// gfx950 bf16 path: direct-to-LDS multi-stage GEMM (gemm2.hpp)
template <int GM, bool AT, bool BT, int EPI, int BM, int BN, int WM, int WN, int ST, int BK, int STO = STORE_DIRECT,
          int XB = 0>
static void run_gemm2(GemmArgs<bf16> p, int64_t tiles_ub, hipStream_t st) {
  if (tiles_ub <= 0) return;
  auto kern = grouped_gemm2<GM, AT, BT, EPI, BM, BN, WM, WN, ST, 1, BK, STO, XB>;
  constexpr int NT = 64 * WM * WN;
  const size_t lds = gemm2_lds_bytes<BM, BN, ST, AT, BT, BK, WM * WN, STO, XB>();
  static std::atomic<int> per_cu[MAX_DEVICES];
  static const char* name = [] {
    static char b[96];
    snprintf(b, sizeof b, "grouped_gemm2<GM=%d,AT=%d,BT=%d,EPI=%d,%dx%d,ST=%d,BK=%d%s>", GM, (int)AT, (int)BT, EPI,
             BM + 32 * XB, BN, ST, BK, XB ? ",XB" : "");
    return b;
  }();
  const int nb = blocks_per_cu(per_cu, (const void*)kern, NT, lds);
  const int64_t resident = (int64_t)nb * device_cus();
  const int grid = (int)std::min<int64_t>(tiles_ub, resident);
  p.chunked = grid >= 8;
  DMOE_LAUNCH_NAMED(name, kern, dim3(grid), dim3(NT), lds, st, p);
}

template <typename E>
static GemmArgs<E> args_m(const int32_t* offsets, const int32_t* tpre, int scale, int N) {
  GemmArgs<E> p{};
  p.offsets = offsets; p.tprefix = tpre; p.tscale = scale; p.groups = N;
  return p;
}

// fp32 tile shapes (register-staged MFMA GEMM of gemm.hpp).  TMR: rows an m-tile holds.
struct CfgF32    { static constexpr int BM = 32, BN = 64, BK = 32, WM = 1, WN = 2, TMR = BM; };
struct CfgDWF32  { static constexpr int BM = 64, BN = 64, BK = 32, WM = 2, WN = 2; };

// bf16 tile shapes of the gemm2 path: many rows per expert -> 256x256 tiles, 8 waves,
// 64-deep k, 2 stages (best of the measured shapes at the wide workload for all three
// operand layouts); few rows -> 32x256 tiles, 4 waves, 4 stages (weight streaming).
// Weight gradients contract over an expert's rows: 64-deep k-steps when experts hold
// many rows, 32-deep ones when they hold few (a k-step past an expert's last row is
// zero-filled in LDS and still multiplied, so with ~16 rows per expert a 64-deep step
// spends three quarters of its MFMA and LDS reads on zeros).
// Weight-gradient tiles write their 128 KiB of output through LDS as whole 128-byte
// lines with the non-temporal hint: the 64 GiB of weight gradients per step then
// stream past the L2 instead of evicting the GEMM's operands from it.
// Many rows per expert: the 256-row tiles take a ninth, shared 32-row block (XB), so an
// m-tile holds up to 288 rows and an expert's rows split evenly over its m-tiles (an
// expert of 512 + 18 rows gets two tiles of 9 and 8 blocks instead of a third tile of
// one block that streams the expert's weights once more).
struct G2Fat     { static constexpr int BM = 256, BN = 256, WM = 4, WN = 2, ST = 2, BK = 64, XB = 1,
                   TMR = BM + 32 * XB; };
struct G2Skinny  { static constexpr int BM = 32, BN = 256, WM = 1, WN = 4, ST = 4, BK = 64, XB = 0, TMR = BM; };
struct G2DW      { static constexpr int BM = 256, BN = 256, WM = 4, WN = 2, ST = 2, BK = 64,
                   STO = STORE_STAGED_NT; };
struct G2DWShort { static constexpr int BM = 256, BN = 256, WM = 4, WN = 2, ST = 4, BK = 32,
                   STO = STORE_STAGED_NT; };

static bool use_fat(const Shape& s) { return s.P >= (int64_t)96 * s.N; }

}  // namespace dmoe
