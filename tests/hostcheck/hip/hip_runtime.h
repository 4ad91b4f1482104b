// Host stand-in for the HIP runtime header, used only by the host address check of the
// grouped GEMM kernels (tests/test_gemm_bounds.py): it lets the kernel source compile for
// the CPU, one thread at a time.  The matrix and cross-lane builtins return data that
// steers no address (zeros or their inputs); barriers and waits are no-ops.
#pragma once
#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <type_traits>
using std::max;
using std::min;
#define __device__
#define __host__
#define __global__
#define __forceinline__ inline
#define __launch_bounds__(...)
#define __shared__
#define __align__(x)
struct uint2 { uint32_t x, y; };
struct uint4 { uint32_t x, y, z, w; };
struct float4 { float x, y, z, w; };
struct hostcheck_dim3 { unsigned x, y, z; };
inline uint2 make_uint2(uint32_t a, uint32_t b) { return {a, b}; }
inline uint4 make_uint4(uint32_t a, uint32_t b, uint32_t c, uint32_t d) { return {a, b, c, d}; }
inline float4 make_float4(float a, float b, float c, float d) { return {a, b, c, d}; }
inline float __uint_as_float(uint32_t u) { float f; std::memcpy(&f, &u, 4); return f; }
inline uint32_t __float_as_uint(float f) { uint32_t u; std::memcpy(&u, &f, 4); return u; }
inline float __expf(float x) { return expf(x); }
template <typename T> inline T __shfl_xor(T v, int, int = 64) { return v; }
inline void __syncthreads() {}
extern thread_local hostcheck_dim3 threadIdx, blockIdx, gridDim, blockDim;
typedef void* hipStream_t;
typedef void* hipEvent_t;
enum { hipSuccess = 0 };
inline int hipEventRecord(hipEvent_t, hipStream_t) { return 0; }
inline int hipGetLastError() { return 0; }
#define hipLaunchKernelGGL(...) ((void)0)
#define __builtin_amdgcn_readfirstlane(x) (x)
#define __builtin_amdgcn_sched_barrier(x) ((void)0)
#define __builtin_amdgcn_sched_group_barrier(x, y, z) ((void)0)
#define __builtin_amdgcn_s_waitcnt(x) ((void)0)
#define __builtin_amdgcn_rcpf(x) (1.0f / (x))
#define __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, x, y, z) (c)
#define __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, x, y, z) (c)
#define __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, x, y, z) (c)
struct hostcheck_pair { uint32_t v[2]; uint32_t operator[](int i) const { return v[i]; } };
inline hostcheck_pair hostcheck_swap(uint32_t a, uint32_t b) { return {{a, b}}; }
#define __builtin_amdgcn_permlane16_swap(a, b, fi, bc) hostcheck_swap((a), (b))
#define __builtin_amdgcn_permlane32_swap(a, b, fi, bc) hostcheck_swap((a), (b))
typedef short hostcheck_s16x4 __attribute__((ext_vector_type(4)));
hostcheck_s16x4 hostcheck_lds_tr(const void* p);
#define __builtin_amdgcn_ds_read_tr16_b64_v4i16(p) hostcheck_lds_tr((const void*)(p))
#define __builtin_nontemporal_store(v, p) (*(p) = (v))
