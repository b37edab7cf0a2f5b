// Achievable-ceiling probes of one MI355X, measured beside the hot path so
// that its roofline fractions can be read against what the device delivers as
// well as against the vendor peaks.  Not part of the hot path's library.
//
// HBM: each wavefront reads whole pieces (for example the 8 KiB a decode unit
// reads per page: a 4 KiB key page and a 4 KiB value page) at given piece
// indices of a large buffer with 16-byte loads (optionally non-temporal, as
// the decode share reads its pages), `inflight` pieces outstanding at a time,
// and folds them into one word per lane (written once, so no load is dead).  MFMA: back-to-back v_mfma_f32_32x32x16_bf16 in independent
// accumulator chains per wavefront.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "dlfp_probe.h"

namespace {

typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

// Piece p of wavefront w is pieces[w * per_wave + p]; a piece of `bytes`
// bytes is read as bytes / 1024 rounds of one 16-byte load per lane, with
// INFLIGHT pieces issued before any is consumed.
template <int INFLIGHT, bool NT>
__global__ __launch_bounds__(256) void hbm_read_kernel(const char* buf, int64_t buf_pieces,
                                                       const int32_t* pieces, int32_t per_wave,
                                                       int32_t piece_bytes, uint32_t* sink) {
  const int lane = threadIdx.x & 63;
  const int64_t wave = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
  const int32_t* my = pieces + wave * per_wave;
  const int rounds = piece_bytes / 1024;
  uint32_t acc = 0;
  for (int p0 = 0; p0 < per_wave; p0 += INFLIGHT) {
    u32x4_t v[INFLIGHT][8];
#pragma unroll
    for (int i = 0; i < INFLIGHT; ++i) {
      const int p = min(p0 + i, per_wave - 1);
      const int64_t idx = min<int64_t>(max(__builtin_amdgcn_readfirstlane(my[p]), 0), buf_pieces - 1);
      const char* base = buf + idx * piece_bytes;
#pragma unroll
      for (int r = 0; r < 8; ++r)
        if (r < rounds) {
          const u32x4_t* src = reinterpret_cast<const u32x4_t*>(base + r * 1024 + 16 * lane);
          v[i][r] = NT ? __builtin_nontemporal_load(src) : *src;
        }
    }
#pragma unroll
    for (int i = 0; i < INFLIGHT; ++i)
#pragma unroll
      for (int r = 0; r < 8; ++r)
        if (r < rounds && p0 + i < per_wave) acc ^= v[i][r][0] ^ v[i][r][1] ^ v[i][r][2] ^ v[i][r][3];
  }
  sink[wave * 64 + lane] = acc;
}

__global__ __launch_bounds__(256) void mfma_kernel(int32_t iters, float* sink) {
  const int lane = threadIdx.x & 63;
  bf16x8_t a, b;
#pragma unroll
  for (int i = 0; i < 8; ++i) {
    a[i] = (__bf16)(0.001f * (lane + i));
    b[i] = (__bf16)(0.002f * (lane - i));
  }
  f32x16_t c0 = {}, c1 = {}, c2 = {}, c3 = {};
  for (int it = 0; it < iters; ++it) {
    c0 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c0, 0, 0, 0);
    c1 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c1, 0, 0, 0);
    c2 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c2, 0, 0, 0);
    c3 = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c3, 0, 0, 0);
  }
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < 16; ++i) s += c0[i] + c1[i] + c2[i] + c3[i];
  sink[(int64_t)blockIdx.x * 256 + threadIdx.x] = s;
}

template <bool NT>
int launch_hbm_read(const char* b, int64_t n, const int32_t* pieces, int32_t waves,
                    int32_t per_wave, int32_t piece_bytes, int32_t inflight, uint32_t* sink,
                    hipStream_t stream) {
  const dim3 grid(waves / 4);
  switch (inflight) {
    case 1: hbm_read_kernel<1, NT><<<grid, 256, 0, stream>>>(b, n, pieces, per_wave, piece_bytes, sink); break;
    case 2: hbm_read_kernel<2, NT><<<grid, 256, 0, stream>>>(b, n, pieces, per_wave, piece_bytes, sink); break;
    case 4: hbm_read_kernel<4, NT><<<grid, 256, 0, stream>>>(b, n, pieces, per_wave, piece_bytes, sink); break;
    default: return -1;
  }
  return 0;
}

}  // namespace

extern "C" int dlfp_probe_hbm_read(const void* buf, int64_t buf_bytes, const int32_t* pieces,
                                   int32_t waves, int32_t per_wave, int32_t piece_bytes,
                                   int32_t inflight, int32_t nontemporal, uint32_t* sink,
                                   hipStream_t stream) {
  if (!buf || !pieces || !sink || waves <= 0 || waves % 4 || per_wave <= 0) return -1;
  if (nontemporal != 0 && nontemporal != 1) return -1;
  if (inflight != 1 && inflight != 2 && inflight != 4) return -1;
  if (piece_bytes < 1024 || piece_bytes > 8192 || piece_bytes % 1024) return -1;
  if (buf_bytes < piece_bytes) return -1;
  (void)hipGetLastError();
  const char* b = static_cast<const char*>(buf);
  const int64_t n = buf_bytes / piece_bytes;
  if (nontemporal)
    launch_hbm_read<true>(b, n, pieces, waves, per_wave, piece_bytes, inflight, sink, stream);
  else
    launch_hbm_read<false>(b, n, pieces, waves, per_wave, piece_bytes, inflight, sink, stream);
  return hipGetLastError() == hipSuccess ? 0 : -4;
}

extern "C" int dlfp_probe_mfma(int32_t workgroups, int32_t iters, float* sink,
                               hipStream_t stream) {
  if (!sink || workgroups <= 0 || iters <= 0) return -1;
  (void)hipGetLastError();
  mfma_kernel<<<workgroups, 256, 0, stream>>>(iters, sink);
  return hipGetLastError() == hipSuccess ? 0 : -4;
}
