// Shared device helpers of libdmoe: element types, bf16 rounding, MFMA wrappers,
// launch checks and the workspace layout.  gfx950 (CDNA4), wave64.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stddef.h>

#include "dmoe.h"

namespace dmoe {

typedef uint16_t bf16;   // bf16 storage (bit pattern)

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

constexpr int KMAX = 8;          // largest k
constexpr int DMAX = 4;          // largest grid dimensionality
constexpr int DM_MAX = 128;      // largest d*M (gate columns)
constexpr int NMAX = 16384;      // largest expert count (LDS histogram)
constexpr int WAVE = 64;

__device__ __forceinline__ float bf2f(bf16 v) { return __uint_as_float((uint32_t)v << 16); }

// fp32 -> bf16, round to nearest even, NaN stays NaN: the gfx950 packed conversion
// v_cvt_pk_bf16_f32 (bit-identical, over every fp32 input, to rounding the bit
// pattern by adding 0x7fff plus the lowest kept bit and quieting NaNs).
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
__device__ __forceinline__ uint32_t f2bf2(float lo, float hi) {
  const f32x2_t v = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2_t));
}
__device__ __forceinline__ bf16 f2bf(float f) { return (bf16)(f2bf2(f, 0.f) & 0xffffu); }

template <typename E> __device__ __forceinline__ float ldf(const E* p);
template <> __device__ __forceinline__ float ldf<float>(const float* p) { return *p; }
template <> __device__ __forceinline__ float ldf<bf16>(const bf16* p) { return bf2f(*p); }

template <typename E> __device__ __forceinline__ E cvt(float v);
template <> __device__ __forceinline__ float cvt<float>(float v) { return v; }
template <> __device__ __forceinline__ bf16 cvt<bf16>(float v) { return f2bf(v); }

// 16-byte vector of elements <-> 16/sizeof(E) floats
template <typename E> struct Vec;
template <> struct Vec<float> {
  static constexpr int N = 4;
  __device__ static void unpack(const uint4& v, float* f) {
    f[0] = __uint_as_float(v.x); f[1] = __uint_as_float(v.y);
    f[2] = __uint_as_float(v.z); f[3] = __uint_as_float(v.w);
  }
  __device__ static uint4 pack(const float* f) {
    return make_uint4(__float_as_uint(f[0]), __float_as_uint(f[1]),
                      __float_as_uint(f[2]), __float_as_uint(f[3]));
  }
};
template <> struct Vec<bf16> {
  static constexpr int N = 8;
  __device__ static void unpack(const uint4& v, float* f) {
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      f[2 * i] = __uint_as_float(w[i] << 16);
      f[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
    }
  }
  __device__ static uint4 pack(const float* f) {
    uint32_t w[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) w[i] = f2bf2(f[2 * i], f[2 * i + 1]);
    return make_uint4(w[0], w[1], w[2], w[3]);
  }
};

// Activations.  GELU is the erf form 0.5 h (1 + erf(h / sqrt 2)).
__device__ __forceinline__ float act_fwd(float h, int act) {
  if (act == DMOE_RELU) return h > 0.f ? h : 0.f;
  return 0.5f * h * (1.f + erff(h * 0.70710678118654752f));
}
// derivative: ReLU' = [h > 0]; GELU' = Phi(h) + h phi(h)
__device__ __forceinline__ float act_bwd(float h, int act) {
  if (act == DMOE_RELU) return h > 0.f ? 1.f : 0.f;
  const float phi = 0.39894228040143268f * __expf(-0.5f * h * h);
  return 0.5f * (1.f + erff(h * 0.70710678118654752f)) + h * phi;
}

// erfc(z) for z >= 0 as t exp(-z^2 + P(t)) with t = 1 / (1 + z/2) and P a degree-9
// polynomial: the Chebyshev-fitted approximation of Numerical Recipes in C (2nd ed.,
// sec. 6.2, "erfcc"), fractional error below 1.2e-7 for every z >= 0 (about 1e-5 when
// evaluated in fp32).  Branch-free, one exponential and one reciprocal.
__device__ __forceinline__ float erfc_pos(float z) {
  const float t = __builtin_amdgcn_rcpf(1.f + 0.5f * z);
  float q = 0.17087277f;
  q = fmaf(q, t, -0.82215223f);
  q = fmaf(q, t, 1.48851587f);
  q = fmaf(q, t, -1.13520398f);
  q = fmaf(q, t, 0.27886807f);
  q = fmaf(q, t, -0.18628806f);
  q = fmaf(q, t, 0.09678418f);
  q = fmaf(q, t, 0.37409196f);
  q = fmaf(q, t, 1.00002368f);
  q = fmaf(q, t, -1.26551223f);
  return t * __expf(q - z * z);
}
// GELU and its derivative through erfc, for the bf16 paths (results are rounded to
// bf16, 2^-9 relative).  1 + erf(h / sqrt 2) = 2 - erfc(|h| / sqrt 2) for h >= 0 and
// erfc(|h| / sqrt 2) for h < 0, which keeps full relative accuracy in the negative tail.
__device__ __forceinline__ float act_fwd_fast(float h, int act) {
  if (act == DMOE_RELU) return h > 0.f ? h : 0.f;
  const float q = erfc_pos(fabsf(h) * 0.70710678118654752f);
  return 0.5f * h * (h >= 0.f ? 2.f - q : q);
}
__device__ __forceinline__ float act_bwd_fast(float h, int act) {
  if (act == DMOE_RELU) return h > 0.f ? 1.f : 0.f;
  const float q = erfc_pos(fabsf(h) * 0.70710678118654752f);
  const float phi = 0.39894228040143268f * __expf(-0.5f * h * h);
  return 0.5f * (h >= 0.f ? 2.f - q : q) + h * phi;
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, WAVE);
  return v;
}

// ----------------------------------------------------------------- host side

struct Shape {
  int64_t T, D, H, N, P, dM;
  int d, M, k, dtype, act, flags;
  size_t esz;   // bytes per element of the layer dtype
};

int check_dims(const dmoe_dims* dims, Shape* s);

// Launch trace (dmoe_trace_begin / dmoe_trace_end): while a trace is active on the
// calling host thread, every kernel an entry point enqueues is followed on its stream by
// a record of the caller's next event, and the kernel's name is noted beside it.
struct TraceState {
  void* const* events;   // hipEvent_t handles, caller-owned
  const char** names;
  int cap, n;
};
extern thread_local TraceState* t_trace;
inline void trace_mark(hipStream_t st, const char* name) {
  TraceState* t = t_trace;
  if (!t) return;
  if (t->n < t->cap) {
    (void)hipEventRecord(reinterpret_cast<hipEvent_t>(t->events[t->n]), st);
    t->names[t->n] = name;
  }
  ++t->n;
}
// Every kernel of the library is enqueued through these: a launch, then its trace mark.
#define DMOE_LAUNCH_NAMED(name, kernel, grid, block, lds, st, ...)          \
  do {                                                                     \
    hipLaunchKernelGGL(kernel, grid, block, lds, st, __VA_ARGS__);         \
    ::dmoe::trace_mark(st, name);                                          \
  } while (0)
#define DMOE_LAUNCH(kernel, grid, block, lds, st, ...) \
  DMOE_LAUNCH_NAMED(#kernel, kernel, grid, block, lds, st, __VA_ARGS__)

inline int launch_status() {
  return hipGetLastError() == hipSuccess ? DMOE_OK : DMOE_EHIP;
}

inline bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

// Workspace regions (byte offsets into the caller's ws buffer).
struct Workspace {
  size_t hist_off, hist_bytes;     // dispatch: per-block expert histograms
  size_t tiles_off, tiles_bytes;   // grouped GEMM: tile prefix [N+1] + per-expert m-tiles
  size_t ds_off, ds_bytes;         // gate backward: dense ds (bf16 hi/lo or fp32)
  size_t part_off, part_bytes;     // gate backward: dWg partial sums per token split
  size_t gq_off, gq_bytes;         // gate forward: [0] count, [GQ_HEAD + i] tokens to recompute
  size_t total;
  int64_t disp_blocks;             // dispatch blocks (pairs per block = DISP_CHUNK)
  int64_t gsplit, gsplit_tokens;   // gate backward token splits
  int64_t ds_ld;                   // ds row stride (elements)
};

constexpr int DISP_CHUNK = 1024;   // pairs per dispatch block
constexpr int GQ_HEAD = 64;        // gate queue: the count sits on its own 256-byte line

Workspace workspace_layout(const Shape& s);

// Zero `bytes` bytes at p on stream st with a kernel (no hipMemsetAsync).
void fill_zero(void* p, size_t bytes, hipStream_t st);

}  // namespace dmoe
