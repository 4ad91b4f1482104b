// Expert feed-forward blocks on the per-expert row groups (the Runtime's batched
// Forward and Backward of Sec. 3.3), as grouped GEMMs on MFMA.
#include <algorithm>

#include "grouped.hpp"

namespace dmoe {

template <typename C>
static void ffn_fwd_bf16(const Shape& s, const int32_t* offsets, const bf16* xp, const bf16* W1,
                         const bf16* b1, const bf16* W2, const bf16* b2, bf16* h, bf16* a, bf16* yp,
                         int32_t* tpre, hipStream_t st) {
  const int N = (int)s.N, D = (int)s.D, H = (int)s.H;
  const int64_t mt_ub = (s.P + C::TMR - 1) / C::TMR + std::min<int64_t>(s.N, s.P);
  DMOE_LAUNCH(tile_plan, dim3(1), dim3(1024), 0, st, offsets, N, C::TMR, tpre);
  {
    const int nt = (H + C::BN - 1) / C::BN;
    GemmArgs<bf16> p = args_m<bf16>(offsets, tpre, nt, N);
    p.A = xp; p.lda = D;
    p.B = W1; p.ldb = D; p.b_gstride = (int64_t)H * D;
    p.C = h; p.ldc = H; p.C2 = a;
    p.bias = b1; p.bias_gstride = H;
    p.N = H; p.K = D; p.act = s.act;
    run_gemm2<GROUP_M, false, false, EPI_BIAS_ACT, C::BM, C::BN, C::WM, C::WN, C::ST, C::BK, STORE_DIRECT, C::XB>(p, mt_ub * nt, st);
  }
  {
    const int nt = (D + C::BN - 1) / C::BN;
    GemmArgs<bf16> p = args_m<bf16>(offsets, tpre, nt, N);
    p.A = a; p.lda = H;
    p.B = W2; p.ldb = H; p.b_gstride = (int64_t)D * H;
    p.C = yp; p.ldc = D;
    p.bias = b2; p.bias_gstride = D;
    p.N = D; p.K = H; p.act = s.act;
    run_gemm2<GROUP_M, false, false, EPI_BIAS, C::BM, C::BN, C::WM, C::WN, C::ST, C::BK, STORE_DIRECT, C::XB>(p, mt_ub * nt, st);
  }
}

// The up-projection of the forward alone (h = x W1^T + b1, a = act(h)), for the
// recompute form of the backward.
template <typename C>
static void ffn_up_bf16(const Shape& s, const int32_t* offsets, const bf16* xp, const bf16* W1, const bf16* b1,
                        bf16* h, bf16* a, int32_t* tpre, hipStream_t st) {
  const int N = (int)s.N, D = (int)s.D, H = (int)s.H;
  const int64_t mt_ub = (s.P + C::TMR - 1) / C::TMR + std::min<int64_t>(s.N, s.P);
  DMOE_LAUNCH(tile_plan, dim3(1), dim3(1024), 0, st, offsets, N, C::TMR, tpre);
  const int nt = (H + C::BN - 1) / C::BN;
  GemmArgs<bf16> p = args_m<bf16>(offsets, tpre, nt, N);
  p.A = xp; p.lda = D;
  p.B = W1; p.ldb = D; p.b_gstride = (int64_t)H * D;
  p.C = h; p.ldc = H; p.C2 = a;
  p.bias = b1; p.bias_gstride = H;
  p.N = H; p.K = D; p.act = s.act;
  run_gemm2<GROUP_M, false, false, EPI_BIAS_ACT, C::BM, C::BN, C::WM, C::WN, C::ST, C::BK, STORE_DIRECT, C::XB>(p, mt_ub * nt, st);
}

template <typename C, typename CW>
static void ffn_bwd_bf16(const Shape& s, const int32_t* offsets, const bf16* xp, const bf16* h,
                         const bf16* a, const bf16* dyp, const bf16* W1, const bf16* W2, bf16* dh, bf16* dxp,
                         bf16* dW1, bf16* db1, bf16* dW2, bf16* db2, int32_t* tpre, hipStream_t st) {
  const int N = (int)s.N, D = (int)s.D, H = (int)s.H;
  const int64_t mt_ub = (s.P + C::TMR - 1) / C::TMR + std::min<int64_t>(s.N, s.P);
  const int64_t active_ub = std::min<int64_t>(s.N, s.P);
  const int32_t* tact = tpre + N + 1;
  DMOE_LAUNCH(tile_plan, dim3(1), dim3(1024), 0, st, offsets, N, C::TMR, tpre);
  {   // dh = (dy W2) * act'(h): W2_e read as (n = h, k = d), N-contiguous
    const int nt = (H + C::BN - 1) / C::BN;
    GemmArgs<bf16> p = args_m<bf16>(offsets, tpre, nt, N);
    p.A = dyp; p.lda = D;
    p.B = W2; p.ldb = H; p.b_gstride = (int64_t)D * H;
    p.C = dh; p.ldc = H; p.aux = h;
    p.N = H; p.K = D; p.act = s.act;
    run_gemm2<GROUP_M, false, true, EPI_DACT, C::BM, C::BN, C::WM, C::WN, C::ST, C::BK, STORE_DIRECT, C::XB>(p, mt_ub * nt, st);
  }
  {   // dW2_e = dy_e^T a_e   [D, H]
    const int mt = (D + CW::BM - 1) / CW::BM, nt = (H + CW::BN - 1) / CW::BN;
    GemmArgs<bf16> p = args_m<bf16>(offsets, tact, mt * nt, N);
    p.A = dyp; p.lda = D;
    p.B = a; p.ldb = H;
    p.C = dW2; p.ldc = H; p.c_gstride = (int64_t)D * H;
    p.M = D; p.N = H; p.act = s.act;
    run_gemm2<GROUP_K, true, true, EPI_STORE, CW::BM, CW::BN, CW::WM, CW::WN, CW::ST, CW::BK, CW::STO>(p, active_ub * mt * nt, st);
  }
  {   // dx_perm = dh W1: W1_e read as (n = d, k = h), N-contiguous
    const int nt = (D + C::BN - 1) / C::BN;
    GemmArgs<bf16> p = args_m<bf16>(offsets, tpre, nt, N);
    p.A = dh; p.lda = H;
    p.B = W1; p.ldb = D; p.b_gstride = (int64_t)H * D;
    p.C = dxp; p.ldc = D;
    p.N = D; p.K = H; p.act = s.act;
    run_gemm2<GROUP_M, false, true, EPI_STORE, C::BM, C::BN, C::WM, C::WN, C::ST, C::BK, STORE_DIRECT, C::XB>(p, mt_ub * nt, st);
  }
  {   // dW1_e = dh_e^T x_e   [H, D]
    const int mt = (H + CW::BM - 1) / CW::BM, nt = (D + CW::BN - 1) / CW::BN;
    GemmArgs<bf16> p = args_m<bf16>(offsets, tact, mt * nt, N);
    p.A = dh; p.lda = H;
    p.B = xp; p.ldb = D;
    p.C = dW1; p.ldc = D; p.c_gstride = (int64_t)H * D;
    p.M = H; p.N = D; p.act = s.act;
    run_gemm2<GROUP_K, true, true, EPI_STORE, CW::BM, CW::BN, CW::WM, CW::WN, CW::ST, CW::BK, CW::STO>(p, active_ub * mt * nt, st);
  }
  DMOE_LAUNCH(segment_colsum<bf16>, dim3((unsigned)((H / 8 + 255) / 256), (unsigned)N), dim3(256), 0,
                     st, dh, (int64_t)H, offsets, H, db1);
  DMOE_LAUNCH(segment_colsum<bf16>, dim3((unsigned)((D / 8 + 255) / 256), (unsigned)N), dim3(256), 0,
                     st, dyp, (int64_t)D, offsets, D, db2);
}

// Backward with the expert parameters updated in place (W <- W - lr dW, b <- b - lr db),
// the gradients never stored.  Each parameter is updated after its last use: dh reads
// W2 before W2's update, dx_perm reads W1 before W1's update.
template <typename C, typename CW>
static void ffn_bwd_sgd_bf16(const Shape& s, const int32_t* offsets, const bf16* xp, const bf16* a,
                             const bf16* dyp, bf16* W1, bf16* b1, bf16* W2, bf16* b2, float lr, const bf16* h,
                             bf16* dh, bf16* dxp, int32_t* tpre, hipStream_t st) {
  const int N = (int)s.N, D = (int)s.D, H = (int)s.H;
  const int64_t mt_ub = (s.P + C::TMR - 1) / C::TMR + std::min<int64_t>(s.N, s.P);
  const int64_t active_ub = std::min<int64_t>(s.N, s.P);
  const int32_t* tact = tpre + N + 1;
  DMOE_LAUNCH(tile_plan, dim3(1), dim3(1024), 0, st, offsets, N, C::TMR, tpre);
  {   // dh = (dy W2) * act'(h)
    const int nt = (H + C::BN - 1) / C::BN;
    GemmArgs<bf16> p = args_m<bf16>(offsets, tpre, nt, N);
    p.A = dyp; p.lda = D;
    p.B = W2; p.ldb = H; p.b_gstride = (int64_t)D * H;
    p.C = dh; p.ldc = H; p.aux = h;
    p.N = H; p.K = D; p.act = s.act;
    run_gemm2<GROUP_M, false, true, EPI_DACT, C::BM, C::BN, C::WM, C::WN, C::ST, C::BK, STORE_DIRECT, C::XB>(p, mt_ub * nt, st);
  }
  {   // W2_e -= lr dy_e^T a_e
    const int mt = (D + CW::BM - 1) / CW::BM, nt = (H + CW::BN - 1) / CW::BN;
    GemmArgs<bf16> p = args_m<bf16>(offsets, tact, mt * nt, N);
    p.A = dyp; p.lda = D;
    p.B = a; p.ldb = H;
    p.C = W2; p.ldc = H; p.c_gstride = (int64_t)D * H;
    p.M = D; p.N = H; p.act = s.act; p.lr = lr;
    run_gemm2<GROUP_K, true, true, EPI_SGD, CW::BM, CW::BN, CW::WM, CW::WN, CW::ST, CW::BK, CW::STO>(p, active_ub * mt * nt, st);
  }
  {   // dx_perm = dh W1
    const int nt = (D + C::BN - 1) / C::BN;
    GemmArgs<bf16> p = args_m<bf16>(offsets, tpre, nt, N);
    p.A = dh; p.lda = H;
    p.B = W1; p.ldb = D; p.b_gstride = (int64_t)H * D;
    p.C = dxp; p.ldc = D;
    p.N = D; p.K = H; p.act = s.act;
    run_gemm2<GROUP_M, false, true, EPI_STORE, C::BM, C::BN, C::WM, C::WN, C::ST, C::BK, STORE_DIRECT, C::XB>(p, mt_ub * nt, st);
  }
  {   // W1_e -= lr dh_e^T x_e
    const int mt = (H + CW::BM - 1) / CW::BM, nt = (D + CW::BN - 1) / CW::BN;
    GemmArgs<bf16> p = args_m<bf16>(offsets, tact, mt * nt, N);
    p.A = dh; p.lda = H;
    p.B = xp; p.ldb = D;
    p.C = W1; p.ldc = D; p.c_gstride = (int64_t)H * D;
    p.M = H; p.N = D; p.act = s.act; p.lr = lr;
    run_gemm2<GROUP_K, true, true, EPI_SGD, CW::BM, CW::BN, CW::WM, CW::WN, CW::ST, CW::BK, CW::STO>(p, active_ub * mt * nt, st);
  }
  DMOE_LAUNCH((segment_colsum<bf16, true>), dim3((unsigned)((H / 8 + 255) / 256), (unsigned)N), dim3(256), 0,
                     st, dh, (int64_t)H, offsets, H, b1, lr);
  DMOE_LAUNCH((segment_colsum<bf16, true>), dim3((unsigned)((D / 8 + 255) / 256), (unsigned)N), dim3(256), 0,
                     st, dyp, (int64_t)D, offsets, D, b2, lr);
}

template <typename E, typename C>
static void ffn_fwd_cfg(const Shape& s, const int32_t* offsets, const E* xp, const E* W1,
                        const E* b1, const E* W2, const E* b2, E* h, E* a, E* yp, int32_t* tpre,
                        hipStream_t st) {
  const int N = (int)s.N, D = (int)s.D, H = (int)s.H;
  const int64_t mt_ub = (s.P + C::TMR - 1) / C::TMR + std::min<int64_t>(s.N, s.P);
  DMOE_LAUNCH(tile_plan, dim3(1), dim3(1024), 0, st, offsets, N, C::TMR, tpre);
  // h = x W1^T + b1, a = act(h)
  {
    const int nt = (H + C::BN - 1) / C::BN;
    GemmArgs<E> p = args_m<E>(offsets, tpre, nt, N);
    p.A = xp; p.lda = D;
    p.B = W1; p.ldb = D; p.b_gstride = (int64_t)H * D;
    p.C = h; p.ldc = H; p.C2 = a;
    p.bias = b1; p.bias_gstride = H;
    p.N = H; p.K = D; p.act = s.act;
    run_gemm<E, GROUP_M, true, EPI_BIAS_ACT, C::BM, C::BN, C::BK, C::WM, C::WN>(p, mt_ub * nt, st);
  }
  // y = a W2^T + b2
  {
    const int nt = (D + C::BN - 1) / C::BN;
    GemmArgs<E> p = args_m<E>(offsets, tpre, nt, N);
    p.A = a; p.lda = H;
    p.B = W2; p.ldb = H; p.b_gstride = (int64_t)D * H;
    p.C = yp; p.ldc = D;
    p.bias = b2; p.bias_gstride = D;
    p.N = D; p.K = H; p.act = s.act;
    run_gemm<E, GROUP_M, true, EPI_BIAS, C::BM, C::BN, C::BK, C::WM, C::WN>(p, mt_ub * nt, st);
  }
}

// SGD: dW1, db1, dW2, db2 are the parameters W1, b1, W2, b2 themselves, updated in
// place (W <- W - lr dW) after their last read: dh reads W2 before W2's update and
// dx_perm reads W1 before W1's update.
template <typename E, typename C, typename CW, bool SGD = false>
static void ffn_bwd_cfg(const Shape& s, const int32_t* offsets, const E* xp, const E* h,
                        const E* a, const E* dyp, const E* W1, const E* W2, E* dh, E* dxp, E* dW1,
                        E* db1, E* dW2, E* db2, int32_t* tpre, hipStream_t st, float lr = 0.f) {
  constexpr int EPI_W = SGD ? EPI_SGD : EPI_STORE;
  const int N = (int)s.N, D = (int)s.D, H = (int)s.H;
  const int64_t mt_ub = (s.P + C::TMR - 1) / C::TMR + std::min<int64_t>(s.N, s.P);
  const int64_t active_ub = std::min<int64_t>(s.N, s.P);
  const int32_t* tact = tpre + N + 1;
  DMOE_LAUNCH(tile_plan, dim3(1), dim3(1024), 0, st, offsets, N, C::TMR, tpre);
  // dh = (dy W2) * act'(h)       B = W2_e viewed as (n = h, k = d): N-contiguous
  {
    const int nt = (H + C::BN - 1) / C::BN;
    GemmArgs<E> p = args_m<E>(offsets, tpre, nt, N);
    p.A = dyp; p.lda = D;
    p.B = W2; p.ldb = H; p.b_gstride = (int64_t)D * H;
    p.C = dh; p.ldc = H; p.aux = h;
    p.N = H; p.K = D; p.act = s.act;
    run_gemm<E, GROUP_M, false, EPI_DACT, C::BM, C::BN, C::BK, C::WM, C::WN>(p, mt_ub * nt, st);
  }
  // dW2_e = dy_e^T a_e   [D, H]
  {
    const int mt = (D + CW::BM - 1) / CW::BM, nt = (H + CW::BN - 1) / CW::BN;
    GemmArgs<E> p = args_m<E>(offsets, tact, mt * nt, N);
    p.A = dyp; p.lda = D;
    p.B = a; p.ldb = H;
    p.C = dW2; p.ldc = H; p.c_gstride = (int64_t)D * H;
    p.M = D; p.N = H; p.act = s.act; p.lr = lr;
    run_gemm<E, GROUP_K, false, EPI_W, CW::BM, CW::BN, CW::BK, CW::WM, CW::WN>(p, active_ub * mt * nt, st);
  }
  // dx_perm = dh W1              B = W1_e viewed as (n = d, k = h): N-contiguous
  {
    const int nt = (D + C::BN - 1) / C::BN;
    GemmArgs<E> p = args_m<E>(offsets, tpre, nt, N);
    p.A = dh; p.lda = H;
    p.B = W1; p.ldb = D; p.b_gstride = (int64_t)H * D;
    p.C = dxp; p.ldc = D;
    p.N = D; p.K = H; p.act = s.act;
    run_gemm<E, GROUP_M, false, EPI_STORE, C::BM, C::BN, C::BK, C::WM, C::WN>(p, mt_ub * nt, st);
  }
  // dW1_e = dh_e^T x_e   [H, D]
  {
    const int mt = (H + CW::BM - 1) / CW::BM, nt = (D + CW::BN - 1) / CW::BN;
    GemmArgs<E> p = args_m<E>(offsets, tact, mt * nt, N);
    p.A = dh; p.lda = H;
    p.B = xp; p.ldb = D;
    p.C = dW1; p.ldc = D; p.c_gstride = (int64_t)H * D;
    p.M = H; p.N = D; p.act = s.act; p.lr = lr;
    run_gemm<E, GROUP_K, false, EPI_W, CW::BM, CW::BN, CW::BK, CW::WM, CW::WN>(p, active_ub * mt * nt, st);
  }
  // bias gradients
  constexpr int VEC = 16 / sizeof(E);
  DMOE_LAUNCH((segment_colsum<E, SGD>), dim3((unsigned)((H / VEC + 255) / 256), (unsigned)N), dim3(256), 0,
                     st, dh, (int64_t)H, offsets, H, db1, lr);
  DMOE_LAUNCH((segment_colsum<E, SGD>), dim3((unsigned)((D / VEC + 255) / 256), (unsigned)N), dim3(256), 0,
                     st, dyp, (int64_t)D, offsets, D, db2, lr);
}

template <typename E, typename C>
static void ffn_up_cfg(const Shape& s, const int32_t* offsets, const E* xp, const E* W1, const E* b1, E* h, E* a,
                       int32_t* tpre, hipStream_t st) {
  const int N = (int)s.N, D = (int)s.D, H = (int)s.H;
  const int64_t mt_ub = (s.P + C::TMR - 1) / C::TMR + std::min<int64_t>(s.N, s.P);
  DMOE_LAUNCH(tile_plan, dim3(1), dim3(1024), 0, st, offsets, N, C::TMR, tpre);
  const int nt = (H + C::BN - 1) / C::BN;
  GemmArgs<E> p = args_m<E>(offsets, tpre, nt, N);
  p.A = xp; p.lda = D;
  p.B = W1; p.ldb = D; p.b_gstride = (int64_t)H * D;
  p.C = h; p.ldc = H; p.C2 = a;
  p.bias = b1; p.bias_gstride = H;
  p.N = H; p.K = D; p.act = s.act;
  run_gemm<E, GROUP_M, true, EPI_BIAS_ACT, C::BM, C::BN, C::BK, C::WM, C::WN>(p, mt_ub * nt, st);
}

// The forward on a tile plan at tpre (2 (N + 1) ints of device memory).
static int ffn_fwd_impl(const Shape& s, const int32_t* offsets, const void* x_perm, const void* W1,
                        const void* b1, const void* W2, const void* b2, void* h, void* a, void* y_perm,
                        int32_t* tpre, hipStream_t st) {
  if (s.dtype == DMOE_BF16) {
    auto c = [](const void* q) { return reinterpret_cast<const bf16*>(q); };
    auto m = [](void* q) { return reinterpret_cast<bf16*>(q); };
    if (use_fat(s))
      ffn_fwd_bf16<G2Fat>(s, offsets, c(x_perm), c(W1), c(b1), c(W2), c(b2), m(h), m(a), m(y_perm), tpre, st);
    else
      ffn_fwd_bf16<G2Skinny>(s, offsets, c(x_perm), c(W1), c(b1), c(W2), c(b2), m(h), m(a), m(y_perm), tpre, st);
  } else {
    auto c = [](const void* q) { return reinterpret_cast<const float*>(q); };
    auto m = [](void* q) { return reinterpret_cast<float*>(q); };
    ffn_fwd_cfg<float, CfgF32>(s, offsets, c(x_perm), c(W1), c(b1), c(W2), c(b2), m(h), m(a), m(y_perm), tpre, st);
  }
  return launch_status();
}

static int ffn_fwd_check(const dmoe_dims* dims, Shape* s, const int32_t* offsets, const void* x_perm, const void* W1,
                         const void* b1, const void* W2, const void* b2, const void* h, const void* a,
                         const void* y_perm) {
  const int rc = check_dims(dims, s);
  if (rc) return rc;
  if (s->T == 0) return DMOE_OK;
  if (!offsets || !x_perm || !W1 || !b1 || !W2 || !b2 || !h || !a || !y_perm) return DMOE_EINVAL;
  for (const void* q : {x_perm, W1, W2, h, a, y_perm})
    if (!aligned16(q)) return DMOE_EUNSUPPORTED;
  return DMOE_OK;
}

// Scratch of dmoe_expert_ffn_fwd_noalloc: the tile plan, 2 (N + 1) ints for N <= NMAX.
// Each device holds its own copy; host code reaches it only through the address
// hipGetSymbolAddress returns on that device (the array's name is no device address
// in host code).
constexpr size_t FFN_SCRATCH_BYTES = ((size_t)2 * (NMAX + 1) * sizeof(int32_t) + 255) & ~(size_t)255;
static __device__ __align__(256) unsigned char scratch[FFN_SCRATCH_BYTES];

// scratch's address on the current device, looked up on the first call there.
static int32_t* scratch_on_device() {
  static std::atomic<void*> addr[MAX_DEVICES];
  const int dev = current_device();
  if (dev < 0) return nullptr;
  void* p = addr[dev].load(std::memory_order_acquire);
  if (!p) {
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) {
      (void)hipGetLastError();
      return nullptr;
    }
    addr[dev].store(p, std::memory_order_release);
  }
  return reinterpret_cast<int32_t*>(p);
}

}  // namespace dmoe

using namespace dmoe;

extern "C" int dmoe_expert_ffn_fwd(const dmoe_dims* dims, const int32_t* offsets, const void* x_perm,
                                   const void* W1, const void* b1, const void* W2, const void* b2,
                                   void* h, void* a, void* y_perm, void* ws, void* stream) {
  Shape s;
  int rc = ffn_fwd_check(dims, &s, offsets, x_perm, W1, b1, W2, b2, h, a, y_perm);
  if (rc || s.T == 0) return rc;
  if (!ws) return DMOE_EINVAL;
  if (!aligned16(ws)) return DMOE_EUNSUPPORTED;
  const Workspace L = workspace_layout(s);
  int32_t* tpre = reinterpret_cast<int32_t*>(reinterpret_cast<unsigned char*>(ws) + L.tiles_off);
  return ffn_fwd_impl(s, offsets, x_perm, W1, b1, W2, b2, h, a, y_perm, tpre, reinterpret_cast<hipStream_t>(stream));
}

extern "C" int dmoe_expert_ffn_fwd_noalloc(const dmoe_dims* dims, const int32_t* offsets, const void* x_perm,
                                           const void* W1, const void* b1, const void* W2, const void* b2,
                                           void* h, void* a, void* y_perm, void* stream) {
  Shape s;
  int rc = ffn_fwd_check(dims, &s, offsets, x_perm, W1, b1, W2, b2, h, a, y_perm);
  if (rc || s.T == 0) return rc;
  if ((size_t)2 * (s.N + 1) * sizeof(int32_t) > FFN_SCRATCH_BYTES) return DMOE_EUNSUPPORTED;
  int32_t* tpre = scratch_on_device();
  if (!tpre) return DMOE_EHIP;
  return ffn_fwd_impl(s, offsets, x_perm, W1, b1, W2, b2, h, a, y_perm, tpre, reinterpret_cast<hipStream_t>(stream));
}

extern "C" int dmoe_expert_ffn_bwd(const dmoe_dims* dims, const int32_t* offsets, const int32_t* counts,
                                   const void* x_perm, const void* h, const void* a, const void* dy_perm,
                                   const void* W1, const void* W2, void* dh, void* dx_perm, void* dW1,
                                   void* db1, void* dW2, void* db2, void* ws, void* stream) {
  (void)counts;
  Shape s;
  int rc = check_dims(dims, &s);
  if (rc) return rc;
  if (s.T == 0) return DMOE_OK;
  if (!offsets || !x_perm || !h || !a || !dy_perm || !W1 || !W2 || !dh || !dx_perm || !dW1 || !db1 ||
      !dW2 || !db2 || !ws)
    return DMOE_EINVAL;
  for (const void* q : {x_perm, h, a, dy_perm, W1, W2, (const void*)dh, (const void*)dx_perm,
                        (const void*)dW1, (const void*)db1, (const void*)dW2, (const void*)db2, (const void*)ws})
    if (!aligned16(q)) return DMOE_EUNSUPPORTED;
  const Workspace L = workspace_layout(s);
  int32_t* tpre = reinterpret_cast<int32_t*>(reinterpret_cast<unsigned char*>(ws) + L.tiles_off);
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  if (s.dtype == DMOE_BF16) {
    auto c = [](const void* q) { return reinterpret_cast<const bf16*>(q); };
    auto m = [](void* q) { return reinterpret_cast<bf16*>(q); };
    if (use_fat(s))
      ffn_bwd_bf16<G2Fat, G2DW>(s, offsets, c(x_perm), c(h), c(a), c(dy_perm), c(W1), c(W2), m(dh),
                                m(dx_perm), m(dW1), m(db1), m(dW2), m(db2), tpre, st);
    else
      ffn_bwd_bf16<G2Skinny, G2DWShort>(s, offsets, c(x_perm), c(h), c(a), c(dy_perm), c(W1), c(W2), m(dh),
                                   m(dx_perm), m(dW1), m(db1), m(dW2), m(db2), tpre, st);
  } else {
    auto c = [](const void* q) { return reinterpret_cast<const float*>(q); };
    auto m = [](void* q) { return reinterpret_cast<float*>(q); };
    ffn_bwd_cfg<float, CfgF32, CfgDWF32>(s, offsets, c(x_perm), c(h), c(a), c(dy_perm), c(W1), c(W2), m(dh),
                                         m(dx_perm), m(dW1), m(db1), m(dW2), m(db2), tpre, st);
  }
  return launch_status();
}

extern "C" int dmoe_expert_ffn_bwd_recompute(const dmoe_dims* dims, const int32_t* offsets, const int32_t* counts,
                                             const void* x_perm, const void* W1, const void* b1, const void* W2,
                                             const void* dy_perm, void* h, void* a, void* dx_perm, void* dW1,
                                             void* db1, void* dW2, void* db2, void* ws, void* stream) {
  Shape s;
  int rc = check_dims(dims, &s);
  if (rc) return rc;
  if (s.T == 0) return DMOE_OK;
  if (!offsets || !x_perm || !W1 || !b1 || !W2 || !dy_perm || !h || !a || !dx_perm || !dW1 || !db1 || !dW2 ||
      !db2 || !ws)
    return DMOE_EINVAL;
  for (const void* q : {x_perm, W1, W2, dy_perm, (const void*)h, (const void*)a, (const void*)dx_perm,
                        (const void*)dW1, (const void*)db1, (const void*)dW2, (const void*)db2, (const void*)ws})
    if (!aligned16(q)) return DMOE_EUNSUPPORTED;
  const Workspace L = workspace_layout(s);
  int32_t* tpre = reinterpret_cast<int32_t*>(reinterpret_cast<unsigned char*>(ws) + L.tiles_off);
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  // 1. recompute the up-projection of the forward into the scratch h and a
  if (s.dtype == DMOE_BF16) {
    auto c = [](const void* q) { return reinterpret_cast<const bf16*>(q); };
    auto m = [](void* q) { return reinterpret_cast<bf16*>(q); };
    if (use_fat(s)) ffn_up_bf16<G2Fat>(s, offsets, c(x_perm), c(W1), c(b1), m(h), m(a), tpre, st);
    else ffn_up_bf16<G2Skinny>(s, offsets, c(x_perm), c(W1), c(b1), m(h), m(a), tpre, st);
  } else {
    auto c = [](const void* q) { return reinterpret_cast<const float*>(q); };
    auto m = [](void* q) { return reinterpret_cast<float*>(q); };
    ffn_up_cfg<float, CfgF32>(s, offsets, c(x_perm), c(W1), c(b1), m(h), m(a), tpre, st);
  }
  // 2. the backward proper, dh written over h
  return dmoe_expert_ffn_bwd(dims, offsets, counts, x_perm, h, a, dy_perm, W1, W2, h, dx_perm, dW1, db1, dW2,
                             db2, ws, stream);
}

extern "C" int dmoe_expert_ffn_bwd_sgd(const dmoe_dims* dims, const int32_t* offsets, const int32_t* counts,
                                       const void* x_perm, const void* h, const void* a, const void* dy_perm,
                                       void* W1, void* b1, void* W2, void* b2, float lr, void* dh, void* dx_perm,
                                       void* ws, void* stream) {
  (void)counts;
  Shape s;
  int rc = check_dims(dims, &s);
  if (rc) return rc;
  if (s.T == 0) return DMOE_OK;
  if (!offsets || !x_perm || !h || !a || !dy_perm || !W1 || !b1 || !W2 || !b2 || !dh || !dx_perm || !ws)
    return DMOE_EINVAL;
  if (!(lr == lr)) return DMOE_EINVAL;                       // NaN step size
  for (const void* q : {x_perm, h, a, dy_perm, (const void*)W1, (const void*)b1, (const void*)W2,
                        (const void*)b2, (const void*)dh, (const void*)dx_perm, (const void*)ws})
    if (!aligned16(q)) return DMOE_EUNSUPPORTED;
  const Workspace L = workspace_layout(s);
  int32_t* tpre = reinterpret_cast<int32_t*>(reinterpret_cast<unsigned char*>(ws) + L.tiles_off);
  hipStream_t st = reinterpret_cast<hipStream_t>(stream);
  if (s.dtype == DMOE_BF16) {
    auto c = [](const void* q) { return reinterpret_cast<const bf16*>(q); };
    auto m = [](void* q) { return reinterpret_cast<bf16*>(q); };
    if (use_fat(s))
      ffn_bwd_sgd_bf16<G2Fat, G2DW>(s, offsets, c(x_perm), c(a), c(dy_perm), m(W1), m(b1), m(W2), m(b2), lr,
                                    c(h), m(dh), m(dx_perm), tpre, st);
    else
      ffn_bwd_sgd_bf16<G2Skinny, G2DWShort>(s, offsets, c(x_perm), c(a), c(dy_perm), m(W1), m(b1), m(W2), m(b2), lr,
                                       c(h), m(dh), m(dx_perm), tpre, st);
  } else {
    auto c = [](const void* q) { return reinterpret_cast<const float*>(q); };
    auto m = [](void* q) { return reinterpret_cast<float*>(q); };
    ffn_bwd_cfg<float, CfgF32, CfgDWF32, true>(s, offsets, c(x_perm), c(h), c(a), c(dy_perm), c(W1), c(W2), m(dh),
                                               m(dx_perm), m(W1), m(b1), m(W2), m(b2), tpre, st, lr);
  }
  return launch_status();
}
