// Paged KV append: write this iteration's new keys and values into their
// pages (the PagedAttention cache write; the cache layout is the one the
// attention launch reads, declared in dlfp.h).
//
// One workgroup of 128 threads serves 16 consecutive packed tokens of one KV
// head.  Keys keep their token-row layout: 16 threads copy one 256-byte row
// with 16-byte loads and stores.  Values go into the transposed page
// [dim][position], token slot t at position vt_pos(t) (slots 4-7 and 8-11
// trade places): thread d gathers dimension d of the 16 tokens (256-byte
// coalesced reads per token) and, when the 16 tokens fill one page in slot
// order -- the common case inside a prefill chunk -- writes its whole 32-byte
// row, so the workgroup stores the 4 KiB page contiguously.  Otherwise each
// token's value lands with a 2-byte store at its position.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "dlfp.h"
#include "dlfp_internal.h"

namespace {

typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));

constexpr int D = DLFP_HEAD_DIM;
constexpr int PAGE = DLFP_PAGE_SIZE;
constexpr int TOK = 16;      // tokens per workgroup
constexpr int THREADS = 128;

// Position of token slot t in a value page row (bits 2 and 3 swap).
__device__ __forceinline__ int vt_pos(int t) { return (t & 3) | ((t & 4) << 1) | ((t & 8) >> 1); }

__global__ __launch_bounds__(THREADS) void kv_append_kernel(
    const uint16_t* __restrict__ k_new, const uint16_t* __restrict__ v_new,
    const int32_t* __restrict__ slots, uint16_t* __restrict__ k_cache,
    uint16_t* __restrict__ v_cache, int num_tokens, int hkv, int64_t num_slots) {
  const int t0 = blockIdx.x * TOK;
  const int h = blockIdx.y;
  const int tid = threadIdx.x;
  const int nt = min(TOK, num_tokens - t0);

  // Every load is issued before any store (one memory round trip): the
  // workgroup's slots, two 16-byte key chunks per thread (tokens tid / 16 and
  // tid / 16 + 8, chunk tid % 16) and the 16 values of dimension d = tid.
  int sl[TOK];
#pragma unroll
  for (int tt = 0; tt < TOK; ++tt) sl[tt] = tt < nt ? slots[t0 + tt] : -1;
  const int c = tid & 15;
  u32x4_t kv[2];
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int tt = (tid >> 4) + 8 * j;
    kv[j] = tt < nt ? *reinterpret_cast<const u32x4_t*>(k_new + ((int64_t)(t0 + tt) * hkv + h) * D + c * 8)
                    : u32x4_t{0u, 0u, 0u, 0u};
  }
  const int d = tid;
  uint16_t vals[TOK];
#pragma unroll
  for (int tt = 0; tt < TOK; ++tt)
    vals[tt] = tt < nt ? v_new[((int64_t)(t0 + tt) * hkv + h) * D + d] : 0;

  // Keys: token rows, 16-byte chunks.
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int tt = (tid >> 4) + 8 * j;
    const int slot = sl[tt];
    if (tt < nt && slot >= 0 && (int64_t)slot < num_slots) {
      const int64_t blk = slot / PAGE, off = slot % PAGE;
      *reinterpret_cast<u32x4_t*>(k_cache + ((blk * hkv + h) * PAGE + off) * D + c * 8) = kv[j];
    }
  }

  // Values: thread d owns dimension d.
  const int s0 = sl[0];
  bool full = nt == TOK && s0 >= 0 && (int64_t)s0 + TOK <= num_slots && (s0 % PAGE) == 0;
#pragma unroll
  for (int tt = 1; tt < TOK; ++tt) full = full && sl[tt] == s0 + tt;
  if (full) {
    const int64_t blk = s0 / PAGE;
    u32x4_t lo, hi;
#pragma unroll
    for (int w = 0; w < 4; ++w) {  // position p holds slot vt_pos(p)
      lo[w] = (uint32_t)vals[vt_pos(2 * w)] | ((uint32_t)vals[vt_pos(2 * w + 1)] << 16);
      hi[w] = (uint32_t)vals[vt_pos(8 + 2 * w)] | ((uint32_t)vals[vt_pos(8 + 2 * w + 1)] << 16);
    }
    u32x4_t* dst = reinterpret_cast<u32x4_t*>(v_cache + ((blk * hkv + h) * D + d) * PAGE);
    dst[0] = lo;
    dst[1] = hi;
  } else {
#pragma unroll
    for (int tt = 0; tt < TOK; ++tt) {
      const int slot = sl[tt];
      if (tt < nt && slot >= 0 && (int64_t)slot < num_slots) {
        const int64_t blk = slot / PAGE, off = slot % PAGE;
        v_cache[((blk * hkv + h) * D + d) * PAGE + vt_pos((int)off)] = vals[tt];
      }
    }
  }
}

}  // namespace

extern "C" int dlfp_kv_append(const dlfp_dims* dims, int32_t num_tokens, const void* k_new,
                              const void* v_new, const int32_t* slot_mapping, void* k_cache,
                              void* v_cache, int32_t num_blocks, hipStream_t stream) {
  int g = 0;
  const int st = dlfp::check_dims(dims, &g);
  if (st != DLFP_OK) return st;
  if (num_tokens < 0 || num_blocks < 0) return DLFP_EINVAL;
  if (num_tokens == 0) return DLFP_OK;
  if (!k_new || !v_new || !slot_mapping || !k_cache || !v_cache) return DLFP_EINVAL;
  (void)hipGetLastError();
  const dim3 grid((num_tokens + TOK - 1) / TOK, dims->num_kv_heads);
  kv_append_kernel<<<grid, THREADS, 0, stream>>>(
      static_cast<const uint16_t*>(k_new), static_cast<const uint16_t*>(v_new), slot_mapping,
      static_cast<uint16_t*>(k_cache), static_cast<uint16_t*>(v_cache), num_tokens,
      dims->num_kv_heads, (int64_t)num_blocks * PAGE);
  return hipGetLastError() == hipSuccess ? DLFP_OK : DLFP_EHIP;
}
