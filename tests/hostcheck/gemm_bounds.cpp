// Host address check of the grouped bf16 GEMM (gemm2.hpp): every thread of every block of
// each launch the layer makes runs the kernel source on the CPU, one thread after another.
// The matrix and cross-lane operations produce data only, which steers no address; global
// buffers and the LDS are allocated at their exact sizes under AddressSanitizer, so an
// access outside them stops the run with its stack.  The launches are set up as the
// layer's forward, backward, fused-SGD and LayerNorm-block entry points set them up, on
// ragged routings (an empty expert, a heavy one, row counts around tile boundaries), for
// both tile families (256 x 256 tiles with the shared 32-row block, and 32 x 256 tiles).
#include <random>
#include <vector>

#include "gemm2.hpp"
#include "g2cfg.hpp"   // the launch helpers' tile shapes G2Fat, G2Skinny, G2DW, G2DWShort

thread_local hostcheck_dim3 threadIdx, blockIdx, gridDim, blockDim;
thread_local char* hostcheck_smem;
namespace dmoe {
void hostcheck_g2l(const void* g, char* l) { std::memcpy(l, g, 16); }
}
hostcheck_s16x4 hostcheck_lds_tr(const void* p) {
  hostcheck_s16x4 v;
  std::memcpy(&v, p, 8);
  return v;
}

using namespace dmoe;

template <typename T>
static T* buf(size_t n) { return static_cast<T*>(std::calloc(n ? n : 1, sizeof(T))); }

// tile plan as the tile_plan kernel writes it: m-tile prefix per expert, then the prefix
// of experts with rows
static std::vector<int32_t> plan_of(const std::vector<int32_t>& off, int N, int TMR) {
  std::vector<int32_t> plan(2 * (N + 1));
  int bm = 0, ba = 0;
  for (int e = 0; e < N; ++e) {
    plan[e] = bm;
    plan[N + 1 + e] = ba;
    const int c = off[e + 1] - off[e];
    bm += (c + TMR - 1) / TMR;
    ba += c > 0;
  }
  plan[N] = bm;
  plan[N + 1 + N] = ba;
  return plan;
}

static long launches = 0;
static size_t dw_short = 0;     // elements taken off the weight-gradient buffer (self-test)

template <int GM, bool AT, bool BT, int EPI, int BM, int BN, int WM, int WN, int ST, int BK, int STO, int XB>
static void run(GemmArgs<bf16> p, int64_t tiles_ub) {
  if (tiles_ub <= 0) return;
  const int NT = 64 * WM * WN;
  const size_t lds = gemm2_lds_bytes<BM, BN, ST, AT, BT, BK, WM * WN, STO, XB>();
  const int grid = (int)std::min<int64_t>(tiles_ub, 256);    // one block per compute unit
  p.chunked = grid >= 8;
  gridDim = {(unsigned)grid, 1, 1};
  blockDim = {(unsigned)NT, 1, 1};
  for (int b = 0; b < grid; ++b)
    for (int t = 0; t < NT; ++t) {
      blockIdx = {(unsigned)b, 0, 0};
      threadIdx = {(unsigned)t, 0, 0};
      hostcheck_smem = static_cast<char*>(std::malloc(lds));
      grouped_gemm2<GM, AT, BT, EPI, BM, BN, WM, WN, ST, 1, BK, STO, XB>(p);
      std::free(hostcheck_smem);
    }
  ++launches;
}

static GemmArgs<bf16> args_m(const std::vector<int32_t>& off, const std::vector<int32_t>& plan, int scale, int N,
                             bool active) {
  GemmArgs<bf16> p{};
  p.offsets = off.data();
  p.tprefix = plan.data() + (active ? N + 1 : 0);
  p.tscale = scale;
  p.groups = N;
  return p;
}

// grouped GEMMs of one Linear layer [n_in -> n_out]: forward with bias (and the
// activation when act), data gradient, weight gradient (stored, or the SGD update)
template <typename C, typename CW>
static void layer(const std::vector<int32_t>& off, int N, int P, int n_in, int n_out, bool act) {
  const auto plan = plan_of(off, N, C::TMR);
  const int64_t mt_ub = (P + C::TMR - 1) / C::TMR + std::min<int64_t>(N, P);
  const int64_t active_ub = std::min<int64_t>(N, P);
  bf16* X = buf<bf16>((size_t)P * n_in);
  bf16* W = buf<bf16>((size_t)N * n_out * n_in);
  bf16* b = buf<bf16>((size_t)N * n_out);
  bf16* Hh = buf<bf16>((size_t)P * n_out);
  bf16* Aa = buf<bf16>((size_t)P * n_out);
  bf16* dY = buf<bf16>((size_t)P * n_out);
  bf16* dX = buf<bf16>((size_t)P * n_in);
  bf16* dW = buf<bf16>((size_t)N * n_out * n_in - dw_short);
  {   // forward: C[rows, n_out] = X W^T + b (h, and a = act(h))
    const int nt = (n_out + C::BN - 1) / C::BN;
    GemmArgs<bf16> p = args_m(off, plan, nt, N, false);
    p.A = X; p.lda = n_in; p.B = W; p.ldb = n_in; p.b_gstride = (int64_t)n_out * n_in;
    p.C = Hh; p.ldc = n_out; p.C2 = Aa; p.bias = b; p.bias_gstride = n_out; p.N = n_out; p.K = n_in;
    if (act) run<GROUP_M, false, false, EPI_BIAS_ACT, C::BM, C::BN, C::WM, C::WN, C::ST, C::BK, STORE_DIRECT, C::XB>(p, mt_ub * nt);
    else run<GROUP_M, false, false, EPI_BIAS, C::BM, C::BN, C::WM, C::WN, C::ST, C::BK, STORE_DIRECT, C::XB>(p, mt_ub * nt);
  }
  {   // data gradient: dX = dY W (W read N-contiguous); with act, times act'(h) of a layer of n_in outputs
    const int nt = (n_in + C::BN - 1) / C::BN;
    GemmArgs<bf16> p = args_m(off, plan, nt, N, false);
    p.A = dY; p.lda = n_out; p.B = W; p.ldb = n_in; p.b_gstride = (int64_t)n_out * n_in;
    p.C = dX; p.ldc = n_in; p.aux = X; p.N = n_in; p.K = n_out;
    if (act) run<GROUP_M, false, true, EPI_DACT, C::BM, C::BN, C::WM, C::WN, C::ST, C::BK, STORE_DIRECT, C::XB>(p, mt_ub * nt);
    else run<GROUP_M, false, true, EPI_STORE, C::BM, C::BN, C::WM, C::WN, C::ST, C::BK, STORE_DIRECT, C::XB>(p, mt_ub * nt);
  }
  {   // weight gradient dW_e = dY_e^T X_e, stored and as the SGD update of W
    const int mt = (n_out + CW::BM - 1) / CW::BM, nt = (n_in + CW::BN - 1) / CW::BN;
    GemmArgs<bf16> p = args_m(off, plan, mt * nt, N, true);
    p.A = dY; p.lda = n_out; p.B = X; p.ldb = n_in;
    p.C = dW; p.ldc = n_in; p.c_gstride = (int64_t)n_out * n_in; p.M = n_out; p.N = n_in;
    run<GROUP_K, true, true, EPI_STORE, CW::BM, CW::BN, CW::WM, CW::WN, CW::ST, CW::BK, CW::STO, 0>(p, active_ub * mt * nt);
    p.C = W; p.lr = 0.5f;
    run<GROUP_K, true, true, EPI_SGD, CW::BM, CW::BN, CW::WM, CW::WN, CW::ST, CW::BK, CW::STO, 0>(p, active_ub * mt * nt);
  }
  std::free(X); std::free(W); std::free(b); std::free(Hh); std::free(Aa);
  std::free(dY); std::free(dX); std::free(dW);
}

// row counts per expert: random around `mean`, expert 1 empty, expert 0 heavy
static std::vector<int32_t> offsets_of(int N, int mean, int spread, unsigned seed) {
  std::mt19937 rng(seed);
  std::vector<int32_t> off(N + 1, 0);
  for (int e = 0; e < N; ++e) {
    int c = mean - spread + (int)(rng() % (2 * spread + 1));
    if (e == 1) c = 0;
    if (e == 0) c = 2 * mean + spread;
    off[e + 1] = off[e] + std::max(c, 0);
  }
  return off;
}

int main(int argc, char** argv) {
  // "short": the weight-gradient buffer is 8 elements short, which the run must report
  if (argc > 1 && std::strcmp(argv[1], "short") == 0) dw_short = 8;
  // (D, H): multiples of 64 as the API requires; one of them not a multiple of 256, so
  // the last column tile and the last m-tile of the weight gradients are partial
  {   // 256 x 256 tiles: experts around 288 rows (8- and 9-block tiles, some 3 m-tiles)
    const int N = 6;
    const auto off = offsets_of(N, 290, 40, 1);
    const int P = off[N];
    layer<G2Fat, G2DW>(off, N, P, 256, 320, true);
    layer<G2Fat, G2DW>(off, N, P, 320, 256, false);
    layer<G2Fat, G2DWShort>(off, N, P, 192, 256, true);
  }
  {   // 32 x 256 tiles: few rows per expert, 32-deep weight-gradient stages
    const int N = 12;
    const auto off = offsets_of(N, 19, 17, 2);
    const int P = off[N];
    layer<G2Skinny, G2DWShort>(off, N, P, 128, 320, true);
    layer<G2Skinny, G2DWShort>(off, N, P, 320, 128, false);
    layer<G2Skinny, G2DW>(off, N, P, 64, 256, false);
  }
  std::printf("gemm bounds: %ld launches checked\n", launches);
  return 0;
}
