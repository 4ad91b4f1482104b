// Host-side validation, workspace layout and error strings of the C ABI.
#include <algorithm>

#include "common.hpp"

namespace dmoe {

int check_dims(const dmoe_dims* dims, Shape* s) {
  if (!dims) return DMOE_EINVAL;
  const dmoe_dims& q = *dims;
  if (q.T < 0 || q.D <= 0 || q.H <= 0 || q.d < 1 || q.M < 1 || q.k < 1) return DMOE_EINVAL;
  if (q.dtype != DMOE_F32 && q.dtype != DMOE_BF16) return DMOE_EINVAL;
  if (q.act != DMOE_RELU && q.act != DMOE_GELU) return DMOE_EINVAL;
  if (q.flags & ~(DMOE_FLAG_GATE_EXACT | DMOE_FLAG_ALIVE_TOPK)) return DMOE_EINVAL;
  if (q.d > DMAX) return DMOE_EUNSUPPORTED;
  int64_t N = 1;
  for (int i = 0; i < q.d; ++i) {
    N *= q.M;
    if (N > NMAX) return DMOE_EUNSUPPORTED;
  }
  if (q.k > N) return DMOE_EINVAL;
  if (q.k > KMAX) return DMOE_EUNSUPPORTED;
  if ((int64_t)q.d * q.M > DM_MAX) return DMOE_EUNSUPPORTED;
  if (q.D % 64 || q.H % 64) return DMOE_EUNSUPPORTED;
  // tile loads address a tile's rows with 32-bit byte offsets (256 rows x ld x 2 bytes)
  if (q.D > (1 << 22) || q.H > (1 << 22)) return DMOE_EUNSUPPORTED;
  // pair and row indices are 32-bit (T * k rows, with headroom for tile rounding)
  if (q.T > (int64_t)0x7fffffff || q.T * q.k > (int64_t)0x7fffffff / 2) return DMOE_EUNSUPPORTED;
  s->T = q.T; s->D = q.D; s->H = q.H; s->N = N; s->P = q.T * q.k; s->dM = (int64_t)q.d * q.M;
  s->d = q.d; s->M = q.M; s->k = q.k; s->dtype = q.dtype; s->act = q.act; s->flags = q.flags;
  s->esz = q.dtype == DMOE_BF16 ? 2 : 4;
  return DMOE_OK;
}

static size_t align256(size_t v) { return (v + 255) & ~(size_t)255; }

Workspace workspace_layout(const Shape& s) {
  Workspace w{};
  size_t off = 0;
  w.disp_blocks = (s.P + DISP_CHUNK - 1) / DISP_CHUNK;
  w.hist_off = off;
  w.hist_bytes = align256((size_t)(w.disp_blocks > 0 ? w.disp_blocks : 1) * s.N * sizeof(int32_t));
  off += w.hist_bytes;
  // token splits of the dWg GEMM: >= 512 tokens each, at most 32 splits
  int64_t split = (s.T + 31) / 32;
  split = split < 512 ? 512 : split;
  split = (split + 31) / 32 * 32;
  w.gsplit_tokens = split;
  w.gsplit = s.T > 0 ? (s.T + split - 1) / split : 0;
  // tile bookkeeping: GEMM tile prefix [N+1] (+ split offsets/prefix of the gate GEMM)
  const int64_t tiles_ints = 2 * (s.N + 1) + 2 * (w.gsplit + 1);
  w.tiles_off = off;
  w.tiles_bytes = align256((size_t)tiles_ints * sizeof(int32_t));
  off += w.tiles_bytes;
  // ds rows: bf16 keeps hi and lo parts; padded to the 16-byte vector width
  if (s.dtype == DMOE_BF16) w.ds_ld = (2 * s.dM + 7) / 8 * 8;
  else w.ds_ld = (s.dM + 3) / 4 * 4;
  w.ds_off = off;
  w.ds_bytes = align256((size_t)s.T * w.ds_ld * s.esz);
  off += w.ds_bytes;
  w.part_off = off;
  w.part_bytes = align256((size_t)w.gsplit * w.ds_ld * s.D * sizeof(float));
  off += w.part_bytes;
  w.gq_off = off;
  w.gq_bytes = align256((size_t)(GQ_HEAD + s.T) * sizeof(int32_t));
  off += w.gq_bytes;
  w.total = off;
  return w;
}

__global__ void fill_zero_kernel(unsigned char* p, size_t bytes) {
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < bytes; i += (size_t)gridDim.x * blockDim.x)
    p[i] = 0;
}

void fill_zero(void* p, size_t bytes, hipStream_t st) {
  if (!bytes) return;
  const size_t blocks = std::min<size_t>((bytes + 255) / 256, 1024);
  DMOE_LAUNCH(fill_zero_kernel, dim3((unsigned)blocks), dim3(256), 0, st,
                     reinterpret_cast<unsigned char*>(p), bytes);
}

thread_local TraceState* t_trace = nullptr;
static thread_local TraceState t_trace_state;

}  // namespace dmoe

using namespace dmoe;

extern "C" int dmoe_trace_begin(void* const* events, const char** names, int capacity) {
  if (capacity < 0 || (capacity > 0 && (!events || !names))) return DMOE_EINVAL;
  t_trace_state = TraceState{events, names, capacity, 0};
  t_trace = &t_trace_state;
  return DMOE_OK;
}

extern "C" int dmoe_trace_end(void) {
  if (!t_trace) return 0;
  const int n = t_trace->n;
  t_trace = nullptr;
  return n;
}

extern "C" size_t dmoe_workspace_bytes(const dmoe_dims* dims) {
  Shape s;
  if (check_dims(dims, &s) != DMOE_OK) return 0;
  return workspace_layout(s).total;
}

extern "C" const char* dmoe_strerror(int code) {
  switch (code) {
    case DMOE_OK: return "ok";
    case DMOE_EINVAL: return "invalid argument (null pointer or bad dims)";
    case DMOE_EUNSUPPORTED: return "unsupported shape or alignment";
    case DMOE_EHIP: return "HIP launch error";
    default: return "unknown error";
  }
}
