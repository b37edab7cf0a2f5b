// Dense projections of one transformer layer's tokens, for the full-iteration
// latency of Eq. 1: the iteration cost the controller observes includes the
// linear layers, whose work grows with the prefill chunk p_t (Sec. 2.1), not
// only the attention.
//
//   out[m][n] = sum_k x[m][k] w[n][k]      (bf16 in, fp32 accumulation)
//
// x is row-major with row stride ldx (elements), w is [n][k] (a linear layer's
// weight as stored: one row per output feature), out row-major with row stride
// ldo.  Workgroup tile: 128 output features x 128 tokens, 64-deep K steps, two
// LDS buffers per operand filled by direct global-to-LDS copies; four
// wavefronts each own 64 x 64 of the tile as 2 x 2 v_mfma_f32_32x32x16_bf16
// accumulators.  The products are computed as out^T = w x^T so that a lane's
// accumulator holds four consecutive features of one token, stored as one
// 8-byte (bf16) or 16-byte (fp32) write.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "dlfp.h"

namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));

constexpr int TILE = 128;      // features (n) and tokens (m) per workgroup
constexpr int KSTEP = 64;      // k per LDS stage
constexpr int ROW_BYTES = KSTEP * 2;               // one 64-deep row of a stage
constexpr int STAGE_BYTES = TILE * ROW_BYTES;      // 16 KiB per operand and stage
constexpr int THREADS = 256;

typedef __attribute__((address_space(3))) char* lds_ptr_t;

// 16 bytes per lane from global memory straight into LDS at lds + 16 lane; the
// caller waits for the vector-memory counter before the data is read.
__device__ __forceinline__ void lds_copy16(const char* src, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off"
               :
               : "v"(src), "s"(lds)
               : "memory", "m0");
}

__device__ __forceinline__ void wait_vmem() {
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
  __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0)
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi) {
  typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
  bf16x2_t v;
  v[0] = (__bf16)lo;
  v[1] = (__bf16)hi;
  return __builtin_bit_cast(uint32_t, v);
}

struct LinArgs {
  const uint16_t* x;
  const uint16_t* w;
  void* out;
  int32_t m, n, k, ldx, ldo, out_f32;
};

// LDS layout of a stage: row r (64 k values, 128 bytes) keeps its 16-byte
// chunk c at position c ^ (r & 7), so the 8 lanes that read the same chunk of
// 8 consecutive rows hit distinct banks.
__global__ __launch_bounds__(THREADS, 2) void linear_kernel(LinArgs a) {
  __shared__ __attribute__((aligned(16))) char smem[4 * STAGE_BYTES];  // W x2, X x2
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int n0 = blockIdx.x * TILE, m0 = blockIdx.y * TILE;
  const int wn = wave >> 1, wm = wave & 1;  // this wave's 64 x 64 quarter

  // Copy assignment: each lane moves 16-byte chunks (4 per operand and stage);
  // LDS chunk q = 256 i + tid sits at row q >> 3, position q & 7, which holds
  // source chunk (q & 7) ^ (row & 7).  Rows past the tokens re-read the last
  // token (their results are not stored).
  const char* wsrc[4];
  const char* xsrc[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int q = 256 * i + tid, r = q >> 3, c = (q & 7) ^ (r & 7);
    wsrc[i] = reinterpret_cast<const char*>(a.w + (int64_t)(n0 + r) * a.k) + 16 * c;
    const int mr = min(m0 + r, a.m - 1);
    xsrc[i] = reinterpret_cast<const char*>(a.x + (int64_t)mr * a.ldx) + 16 * c;
  }
  const uint32_t lds0 = (uint32_t)(uintptr_t)(lds_ptr_t)smem;
  auto issue = [&](int ks, int buf) {
    const int koff = ks * KSTEP * 2;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const uint32_t dst = lds0 + buf * STAGE_BYTES + (256 * i + wave * 64) * 16;
      lds_copy16(wsrc[i] + koff, __builtin_amdgcn_readfirstlane(dst));
      lds_copy16(xsrc[i] + koff, __builtin_amdgcn_readfirstlane(dst + 2 * STAGE_BYTES));
    }
  };

  f32x16_t acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = f32x16_t{};

  // Operand reads: lane l takes row (l % 32) of a 32-row block and k
  // 8 (l / 32) .. + 8 of each 16-deep product.
  const int lr = lane & 31, lh = lane >> 5;
  const int nsteps = a.k / KSTEP;
  issue(0, 0);
  wait_vmem();
  __syncthreads();
  for (int ks = 0; ks < nsteps; ++ks) {
    const int buf = ks & 1;
    if (ks + 1 < nsteps) issue(ks + 1, buf ^ 1);
    const char* wl = smem + buf * STAGE_BYTES;
    const char* xl = smem + (2 + buf) * STAGE_BYTES;
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      const int c = 2 * kk + lh;
      bf16x8_t wf[2], xf[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        const int rw = 64 * wn + 32 * i + lr, rx = 64 * wm + 32 * i + lr;
        wf[i] = *reinterpret_cast<const bf16x8_t*>(wl + rw * ROW_BYTES + ((c ^ (rw & 7)) << 4));
        xf[i] = *reinterpret_cast<const bf16x8_t*>(xl + rx * ROW_BYTES + ((c ^ (rx & 7)) << 4));
      }
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wf[i], xf[j], acc[i][j], 0, 0, 0);
    }
    wait_vmem();      // the next stage has landed
    __syncthreads();  // and every wave is done with this one
  }

  // acc[i][j][r] = out^T[feature 64 wn + 32 i + 8 (r / 4) + 4 lh + r % 4][token 64 wm + 32 j + lr]
#pragma unroll
  for (int j = 0; j < 2; ++j) {
    const int m = m0 + 64 * wm + 32 * j + lr;
    if (m >= a.m) continue;
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        const int n = n0 + 64 * wn + 32 * i + 8 * g + 4 * lh;
        const f32x4_t v = {acc[i][j][4 * g], acc[i][j][4 * g + 1], acc[i][j][4 * g + 2],
                           acc[i][j][4 * g + 3]};
        const int64_t e = (int64_t)m * a.ldo + n;
        if (a.out_f32)
          *reinterpret_cast<f32x4_t*>(static_cast<float*>(a.out) + e) = v;
        else
          *reinterpret_cast<u32x2_t*>(static_cast<uint16_t*>(a.out) + e) =
              u32x2_t{pack_bf16(v[0], v[1]), pack_bf16(v[2], v[3])};
      }
  }
}

}  // namespace

extern "C" int dlfp_linear_bf16(int32_t m, int32_t n, int32_t k, const void* x, int32_t ldx,
                                const void* w, void* out, int32_t ldo, int32_t out_dtype,
                                hipStream_t stream) {
  if (m < 0 || n <= 0 || k <= 0) return DLFP_EINVAL;
  if (out_dtype != 0 && out_dtype != 1) return DLFP_EINVAL;
  if (n % TILE || k % KSTEP) return DLFP_EUNSUPPORTED;
  if (ldx < k || ldo < n || ldx % 8 || ldo % 4) return DLFP_EINVAL;
  if (m == 0) return DLFP_OK;
  if (!x || !w || !out) return DLFP_EINVAL;
  if ((reinterpret_cast<uintptr_t>(x) | reinterpret_cast<uintptr_t>(w)) & 15) return DLFP_EINVAL;
  if (reinterpret_cast<uintptr_t>(out) & (out_dtype ? 15 : 7)) return DLFP_EINVAL;
  LinArgs a{static_cast<const uint16_t*>(x), static_cast<const uint16_t*>(w), out, m, n, k,
            ldx, ldo, out_dtype};
  const dim3 grid(n / TILE, (m + TILE - 1) / TILE);
  (void)hipGetLastError();
  linear_kernel<<<grid, THREADS, 0, stream>>>(a);
  return hipGetLastError() == hipSuccess ? DLFP_OK : DLFP_EHIP;
}
