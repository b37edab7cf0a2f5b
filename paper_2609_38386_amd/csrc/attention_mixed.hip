// Single-launch paged attention for one mixed continuous-batching iteration:
// the decode share (one query token per decoding request) and the prefill
// share (a chunk of prompt tokens, causal over the prompt's cached prefix plus
// the chunk) of Eq. 1, Sec. 2.1, served by one grid.
//
// Grid: the work list's prefill units first, one 256-thread workgroup each,
// then decode units, four per workgroup (one per wavefront).
//
// Prefill unit = (sequence, KV head, tile of 128 query rows, key split).
// Rows are the tile's tokens x the g query heads sharing the KV head, so each
// K/V tile staged in LDS serves all g heads (grouped-query sharing in LDS).
// Each wavefront owns 32 rows and computes, per 64-key tile,
//   S^T = K Q^T        (v_mfma_f32_32x32x16_bf16, fp32 accumulation)
//   online softmax     (exp2 domain; each lane owns one row, so row max and
//                       sum need only one exchange with lane ^ 32)
//   O^T += V^T P^T     (P rounded to bf16; V pages are stored transposed, so
//                       the operand is read straight from LDS)
// Working with S^T and O^T keeps every row statistic lane-local, and the
// accumulator layout of S^T is already the B-operand layout of the PV
// product, so P never leaves registers.  K/V tiles are double-buffered in LDS
// (one barrier per tile), with XOR swizzles that keep the 16 lanes of each
// LDS access phase on distinct banks.
//
// Decode unit = (sequence, KV head, key split), one wavefront.  Memory-bound:
// each 16-token page of K and V (8 KiB) is fetched with fully coalesced,
// non-temporal 16-byte loads one page ahead, staged in the wave's LDS slice,
// and consumed by VALU bf16 dot products (v_dot2 with fp32 accumulation; with
// grouped heads, g >= 2, by 16x16 MFMA instead).  Eight lanes share a key (16
// dims each) and sum their partial dot products with DPP; the per-head row
// max uses DPP and wavefront shuffles; probabilities are handed to the PV
// lanes through LDS, and each lane owns two output dims.
//
// Split-K: a unit whose rows are split over several key ranges writes
// (unnormalised O, running max, running sum) to its workspace slot, releases,
// and bumps its group's counter; the last arriver acquires and merges all
// splits in split-index order (deterministic), writes the output and resets
// the counter to zero for the next launch.
//
// The same kernel, instantiated with APP, also writes the iteration's new
// keys and values into the cache (the append and the attention in one
// launch): a decode unit takes its own new token from k_new / v_new into its
// staged last page and stores it to its slot; leading append workgroups write
// the prompt tokens, and prefill units wait for them before loading a page
// that holds a new token.  Instantiated with MIXED (a launch with both
// shares), the prefill tile loop issues its QK products in the order that
// suits a wavefront sharing its SIMD with a decode wavefront.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>
#include <mutex>
#include <type_traits>

#include "dlfp.h"
#include "dlfp_internal.h"

namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x2_t __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4_t __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2_t __attribute__((ext_vector_type(2)));

constexpr int D = DLFP_HEAD_DIM;
constexpr int PAGE = DLFP_PAGE_SIZE;
constexpr int PAGE_ELEMS = PAGE * D;          // bf16 elements per (block, head) page
constexpr int KV_TILE = 64;                   // keys per prefill tile (4 pages)
constexpr int THREADS = 256;
constexpr int PRE_PTAB = DLFP_MAX_PREFILL_UNIT_KEYS / PAGE;  // block ids of one prefill unit
constexpr int PRE_LDS = 4 * KV_TILE * D * 2 + PRE_PTAB * 4;  // 64 KiB of K/V tiles + 8 KiB
constexpr int DEC_PTAB = DLFP_MAX_DECODE_UNIT_KEYS / PAGE;   // block ids of one decode unit
// Per decode wave: two slots of (K page, V page), probability buffer, block
// ids, and (for g = 8) the query of the group.
constexpr int DEC_Q_LDS = 8 * D * 2;
constexpr int DEC_PAGE_SLOT = 2 * PAGE_ELEMS * 2;  // K and V page, 8 KiB
constexpr int DEC_WAVE_LDS = 2 * DEC_PAGE_SLOT + 16 * 16 * 2 + DEC_PTAB * 4 + DEC_Q_LDS;
constexpr int LDS_BYTES = PRE_LDS > 4 * DEC_WAVE_LDS ? PRE_LDS : 4 * DEC_WAVE_LDS;
// Two workgroups per CU (160 KiB of LDS).
static_assert(2 * (LDS_BYTES + 16) <= 160 * 1024, "two workgroups must share a CU");
constexpr float NEG_BIG = -1.0e30f;
constexpr float LOG2E = 1.4426950408889634f;

static_assert(4 * DEC_WAVE_LDS <= LDS_BYTES, "decode slices must fit the shared buffer");

struct Args {
  const int32_t* work;
  const int32_t* block_table;
  const uint16_t* q;
  const uint16_t* kc;
  const uint16_t* vc;
  void* out;
  float* ws;
  int32_t max_blocks;
  int32_t num_blocks;
  int32_t hq;
  int32_t hkv;
  int32_t num_units;
  int32_t num_prefill;
  int32_t out_f32;
  int32_t decode_waves;  // wavefronts of the decode workgroups of this launch
  int32_t decode_static; // decode units handed out by position, the rest by queue
  int32_t lead;          // prefill workgroups before the first decode workgroup
  int32_t decode_lead;   // decode workgroups before the remaining prefill ones
  int32_t deep;          // decode wavefronts keep two pages in flight
  float scale_log2;      // softmax scale * log2(e)
  // Append launches only: this iteration's keys and values [tokens][hkv][128],
  // the leading workgroups that write the append records stored after the
  // units, and the prefill units that wait for them.
  const uint16_t* k_new;
  const uint16_t* v_new;
  int32_t app_wgs;
  int32_t num_append;
  int32_t num_waiting;
};

__device__ __forceinline__ float dot2(uint32_t a, uint32_t b, float c) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a),
                                         __builtin_bit_cast(bf16x2_t, b), c, false);
}

__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi) {
  bf16x2_t v;
  v[0] = (__bf16)lo;
  v[1] = (__bf16)hi;
  return __builtin_bit_cast(uint32_t, v);
}

__device__ __forceinline__ float fexp2(float x) { return __builtin_amdgcn_exp2f(x); }

template <int CTRL>
__device__ __forceinline__ float dpp(float x) {
  return __builtin_bit_cast(
      float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, x), CTRL, 0xF, 0xF, false));
}
constexpr int DPP_XOR1 = 0xB1;         // quad_perm [1,0,3,2]
constexpr int DPP_XOR2 = 0x4E;         // quad_perm [2,3,0,1]
constexpr int DPP_HALF_MIRROR = 0x141; // lane i <-> 7 - i within 8 lanes
constexpr int DPP_ROR8 = 0x128;        // rotate a 16-lane row by 8

__device__ __forceinline__ float shfl_xor(float x, int m) { return __shfl_xor(x, m); }

// Combine a value with the one of lane ^ 16 (or lane ^ 32) by the gfx950
// permlane swaps (VALU, no LDS round trip): swapping two copies of a value
// leaves the lane's own value in one register and its partner's in the
// other.  Written as assembly because the compiler reads both results of
// the swap builtin from one register, losing the partner's value.
__device__ __forceinline__ void swap16(float& a, float& b) {
  asm volatile("s_nop 1\n\tv_permlane16_swap_b32 %0, %1" : "+v"(a), "+v"(b));
}
__device__ __forceinline__ void swap32(float& a, float& b) {
  asm volatile("s_nop 1\n\tv_permlane32_swap_b32 %0, %1" : "+v"(a), "+v"(b));
}
__device__ __forceinline__ float max_xor16(float x) {
  float a = x, b = x;
  swap16(a, b);
  return fmaxf(a, b);
}
__device__ __forceinline__ float max_xor32(float x) {
  float a = x, b = x;
  swap32(a, b);
  return fmaxf(a, b);
}
__device__ __forceinline__ float sum_xor16(float x) {
  float a = x, b = x;
  swap16(a, b);
  return a + b;
}
__device__ __forceinline__ float sum_xor32(float x) {
  float a = x, b = x;
  swap32(a, b);
  return a + b;
}

__device__ __forceinline__ int uniform(int x) { return __builtin_amdgcn_readfirstlane(x); }

// Work records are read-only for the launch: read through the constant
// address space, so that a wave-uniform record comes in with scalar loads
// (one round trip for all its fields).
typedef const __attribute__((address_space(4))) int32_t* record_ptr;
__device__ __forceinline__ record_ptr as_record(const int32_t* p) {
  const uint64_t v = reinterpret_cast<uint64_t>(p);
  const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)v);
  const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(v >> 32));
  return (record_ptr)(((uint64_t)hi << 32) | lo);
}

// Lanes of one wavefront hand data to each other through LDS.  The hardware
// runs a wave's LDS operations in order; this keeps the compiler from moving a
// lane's LDS accesses across the hand-off (it reasons per lane, so a store to
// an address the lane itself never reads would otherwise be free to move).
__device__ __forceinline__ void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

__device__ __forceinline__ int* group_counter_ptr(float* ws, int grp) {
  return reinterpret_cast<int*>(reinterpret_cast<char*>(ws) + DLFP_WORKSPACE_HEADER) + grp;
}

// Header words of the workspace: the decode queue's next ticket and the
// count of decode wavefronts that found it empty.
__device__ __forceinline__ int* header_word(float* ws, int i) { return reinterpret_cast<int*>(ws) + i; }
constexpr int HDR_TICKET = DLFP_WORKSPACE_TICKET_WORD;
constexpr int HDR_DONE = DLFP_WORKSPACE_DONE_WORD;
// Append launches: append wavefronts finished, waiting prefill units finished.
constexpr int HDR_APPEND = DLFP_WORKSPACE_APPEND_WORD;
constexpr int HDR_WAITED = DLFP_WORKSPACE_WAITED_WORD;

// Error word values: 1 = a block id outside the pool, 2 = a wait for the
// append records ran out.
__device__ __forceinline__ void raise_error(float* ws, int code = 1) {
  __hip_atomic_store(reinterpret_cast<int*>(ws), code, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Append launches.  A prefill unit polls the count of finished append
// workgroups (device-coherent loads, so a stale L2 line is never returned)
// until all have counted themselves; the append workgroups come first in the
// grid and wait for nothing, so they are dispatched before any waiting unit
// and the count is reached.  The poll is bounded all the same: after about
// a second it raises error 2 and goes on.  A waiting unit counts itself on
// a second word once its loop is done (it never polls again); the last one
// zeroes both words for the next launch.  No page that holds a new token is
// read before the wait, so no XCD's L2 holds an old copy of one.
constexpr int APPEND_SPIN_LIMIT = 1 << 20;

__device__ __forceinline__ void wait_for_appends(const Args& a) {
  const int* done = header_word(a.ws, HDR_APPEND);
  const int need = a.app_wgs;
  for (int spins = 0;; ++spins) {
    const int n = uniform(__hip_atomic_load(done, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT));
    if (n >= need) break;
    if (spins == APPEND_SPIN_LIMIT) {
      if ((threadIdx.x & 63) == 0) raise_error(a.ws, 2);
      break;
    }
    __builtin_amdgcn_s_sleep(8);
  }
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

// Split-K partial results cross workgroups (and XCDs, whose L2s are not
// coherent with each other).  They are written with device-coherent stores
// (the sc1 policy: written through to the device coherence point) and read
// back with device-coherent loads (which do not return stale L2 lines), both
// through a buffer resource bounded to the group's slots.  Before a unit
// bumps its group counter it waits until all its vector-memory operations,
// stores included, have completed; the last arriver issues its loads only
// after the counter read has returned.  This orders the exchange without
// writing back or invalidating whole L2 caches per unit.
constexpr int CPOL_SC1 = 16;  // cache-policy bit: coherent at device scope

struct Slots {
  __amdgpu_buffer_rsrc_t r;
};

__device__ __forceinline__ Slots group_slots(float* ws, int group_off, int nsplits,
                                             int slot_floats) {
  return Slots{__builtin_amdgcn_make_buffer_rsrc(ws + group_off, 0, nsplits * slot_floats * 4,
                                                 0x00020000)};
}
__device__ __forceinline__ void pstore4(Slots s, int float_off, f32x4_t v) {
  __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4_t, v), s.r, float_off * 4, 0,
                                         CPOL_SC1);
}
__device__ __forceinline__ void pstore2(Slots s, int float_off, f32x2_t v) {
  __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(u32x2_t, v), s.r, float_off * 4, 0,
                                        CPOL_SC1);
}
__device__ __forceinline__ void pstore1(Slots s, int float_off, float v) {
  __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, v), s.r, float_off * 4, 0,
                                        CPOL_SC1);
}
__device__ __forceinline__ f32x4_t pload4(Slots s, int float_off) {
  return __builtin_bit_cast(f32x4_t,
                            __builtin_amdgcn_raw_buffer_load_b128(s.r, float_off * 4, 0, CPOL_SC1));
}
__device__ __forceinline__ f32x2_t pload2(Slots s, int float_off) {
  return __builtin_bit_cast(f32x2_t,
                            __builtin_amdgcn_raw_buffer_load_b64(s.r, float_off * 4, 0, CPOL_SC1));
}
__device__ __forceinline__ float pload1(Slots s, int float_off) {
  return __builtin_bit_cast(float,
                            __builtin_amdgcn_raw_buffer_load_b32(s.r, float_off * 4, 0, CPOL_SC1));
}
// Floats per partial slot: O (rows x 128), m[rows], l[rows], padded to 256 bytes.
__device__ __forceinline__ int slot_floats_for(int rows) {
  return (rows * (D + 2) + 63) / 64 * 64;
}
// Wait for every outstanding vector-memory operation of this wave (on gfx9 the
// vector-memory counter covers stores) and keep the compiler from moving
// memory operations across the wait.
__device__ __forceinline__ void wait_memory_complete() {
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
  __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0), expcnt and lgkmcnt unconstrained
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
}
__device__ __forceinline__ int arrive(float* ws, int grp) {
  return __hip_atomic_fetch_add(group_counter_ptr(ws, grp), 1, __ATOMIC_RELAXED,
                                __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ int* group_counter(float* ws, int grp) {
  return group_counter_ptr(ws, grp);
}

// Workgroups are dealt round-robin over the 8 XCDs; map them so that each XCD
// gets a contiguous range of prefill units (same KV head -> same L2).
__device__ __forceinline__ int xcd_remap(int b, int n) {
  const int x = b & 7, i = b >> 3;
  const int per = n >> 3, rem = n & 7;
  return x * per + min(x, rem) + i;
}

// Store 4 consecutive output values of one row.
__device__ __forceinline__ void store4(const Args& a, int64_t elem, float v0, float v1, float v2,
                                       float v3) {
  if (a.out_f32) {
    f32x4_t v = {v0, v1, v2, v3};
    *reinterpret_cast<f32x4_t*>(static_cast<float*>(a.out) + elem) = v;
  } else {
    u32x2_t v = {pack_bf16(v0, v1), pack_bf16(v2, v3)};
    *reinterpret_cast<u32x2_t*>(static_cast<uint16_t*>(a.out) + elem) = v;
  }
}

__device__ __forceinline__ void store2(const Args& a, int64_t elem, float v0, float v1) {
  if (a.out_f32) {
    f32x2_t v = {v0, v1};
    *reinterpret_cast<f32x2_t*>(static_cast<float*>(a.out) + elem) = v;
  } else {
    *reinterpret_cast<uint32_t*>(static_cast<uint16_t*>(a.out) + elem) = pack_bf16(v0, v1);
  }
}

// ---------------------------------------------------------------- prefill

// Prefill LDS map: K tiles in two slots at 0 and 16 KiB, V^T tiles in two
// slots at 32 and 48 KiB, the unit's block ids from 64 KiB.
constexpr int TILE_BYTES = KV_TILE * D * 2;  // 16 KiB: 64 keys of K, or of V^T
constexpr int V_BASE = 2 * TILE_BYTES;
constexpr int PTAB_BASE = 4 * TILE_BYTES;
// A running row maximum is only raised once a tile's maximum exceeds it by
// more than this many powers of two, so probabilities stay below 2^8 and the
// accumulators are rescaled rarely (the final division by the row sum makes
// the result independent of the reference maximum).
constexpr float RESCALE_LOG2 = 8.f;

// V^T rows (dims) store their two 16-byte halves swapped when bits 2 and 3
// of the dim differ; 8 (or 16) consecutive dims then cover every LDS bank
// once for each half.
__device__ __forceinline__ int vt_swz(int d) { return ((d >> 2) ^ (d >> 3)) & 1; }

// Position of token slot t inside a V^T row of the cache: slots 4-7 and 8-11
// trade places (bits 2 and 3 swap), matching the key order of the
// S^T accumulator rows that become the PV operand.
__device__ __forceinline__ int vt_pos(int t) { return (t & 3) | ((t & 4) << 1) | ((t & 8) >> 1); }

typedef __attribute__((address_space(3))) char* lds_ptr_t;
// One 16-byte piece per lane, global to LDS without registers: lane l's piece
// lands at LDS byte address lds + 16 l (lds is wave-uniform).  Completion is
// counted by the vector-memory counter; the caller waits for it explicitly
// (wait_memory_complete) before the barrier that publishes the tile.  The
// copy is written as assembly so that the compiler, which cannot tell the
// ring slots apart, does not wait for it before every LDS read.
__device__ __forceinline__ void lds_copy16(const char* src, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off"
               :
               : "v"(src), "s"(lds)
               : "memory", "m0");
}
// The same copy marked non-temporal, for the decode share's pages: each is
// read once per launch, so streaming them past the caches keeps the prefill
// share's K/V tiles (read by many query tiles) resident in L2 and raises the
// decode share's own HBM rate (Qwen3-32B decode-only 5.91 -> 6.49 TB/s).
__device__ __forceinline__ void lds_copy16_nt(const char* src, uint32_t lds) {
  asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off nt"
               :
               : "v"(src), "s"(lds)
               : "memory", "m0");
}
__device__ __forceinline__ uint32_t lds_addr(char* p) {
  return (uint32_t)(uintptr_t)(lds_ptr_t)p;
}

// Keep the elements of a 16-bit-element vector whose key index is below
// limit; key_of(e) gives element e's key.
template <typename F>
__device__ __forceinline__ u32x4_t mask_elems(u32x4_t v, int limit, F key_of) {
#pragma unroll
  for (int w = 0; w < 4; ++w) {
    const uint32_t lo = key_of(2 * w) < limit ? 0x0000FFFFu : 0u;
    const uint32_t hi = key_of(2 * w + 1) < limit ? 0xFFFF0000u : 0u;
    v[w] &= (lo | hi);
  }
  return v;
}

// Last arriver's merge of a prefill group: every split's (O, m, l) in split
// order with an online rescale.  TPR threads per row; a row's 128 values are
// 32 four-float pieces (chunk c = piece / 2, half = piece % 2 of the partial
// layout), and the thread with index sub in its row takes pieces
// sub + TPR i.  The loads of NB splits (pieces, maxima and sums) are issued
// before any is consumed, so a batch costs about one memory round trip; NB is
// chosen so that a batch holds about 136 registers.  Every load instruction
// of a wavefront reads whole contiguous runs of the partial layout.
template <int G, int TPR>
__device__ __forceinline__ void prefill_merge(const Args& a, const Slots sl, int slot_floats,
                                              int nsplits, int rows, int row0, int kh) {
  constexpr int NP = 32 / TPR;             // pieces per thread
  constexpr int PP = NP < 8 ? NP : 8;      // pieces per pass
  constexpr int PASSES = NP / PP;
  constexpr int NB = 32 / PP;              // splits per batch
  const int tid = threadIdx.x;
  if (tid >= TPR * rows) return;
  const int row = tid / TPR, sub = tid % TPR;
  const int64_t orow = ((int64_t)(row0 + row / G) * a.hq + kh * G + row % G) * D;
  for (int pass = 0; pass < PASSES; ++pass) {
    float M = NEG_BIG, lsum = 0.f;
    f32x4_t acc[PP];
#pragma unroll
    for (int i = 0; i < PP; ++i) acc[i] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    for (int j = 0; j < nsplits; j += NB) {
      float mj[NB], lj[NB];
      f32x4_t x[NB][PP];
#pragma unroll
      for (int u = 0; u < NB; ++u) {
        const int b = min(j + u, nsplits - 1) * slot_floats;
        mj[u] = pload1(sl, b + rows * D + row);
        lj[u] = pload1(sl, b + rows * D + rows + row);
#pragma unroll
        for (int i = 0; i < PP; ++i) {
          const int piece = sub + TPR * (pass * PP + i);
          x[u][i] = pload4(sl, b + (((piece >> 1) * rows + row) * 8 + 4 * (piece & 1)));
        }
      }
      float mn = M;
#pragma unroll
      for (int u = 0; u < NB; ++u)
        if (j + u < nsplits) mn = fmaxf(mn, mj[u]);
      const float rs = fexp2(M - mn);
      M = mn;
      lsum *= rs;
#pragma unroll
      for (int i = 0; i < PP; ++i) acc[i] *= rs;
#pragma unroll
      for (int u = 0; u < NB; ++u) {
        const float w = j + u < nsplits ? fexp2(mj[u] - mn) : 0.f;
        lsum += w * lj[u];
#pragma unroll
        for (int i = 0; i < PP; ++i) acc[i] += w * x[u][i];
      }
    }
    const float inv = 1.f / lsum;
#pragma unroll
    for (int i = 0; i < PP; ++i) {
      // piece -> chunk c = 4 mb + g4 and half h -> dims 32 mb + 8 g4 + 4 h
      const int piece = sub + TPR * (pass * PP + i);
      const int c = piece >> 1;
      const int dim = 32 * (c >> 2) + 8 * (c & 3) + 4 * (piece & 1);
      store4(a, orow + dim, acc[i][0] * inv, acc[i][1] * inv, acc[i][2] * inv, acc[i][3] * inv);
    }
  }
}

// MIXED: the launch also has decode units (the QK products' issue order below).
template <int G, bool APP, bool MIXED>
__device__ void prefill_unit(const Args& a, const int32_t* it, char* smem, int* flag) {
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int col = lane & 31, hi = lane >> 5;
  const int s = it[DLFP_W_SEQ], kh = it[DLFP_W_KVHEAD];
  const int t0 = it[DLFP_W_QTOK0], nt = it[DLFP_W_QNTOK];
  const int kb = it[DLFP_W_KVBEGIN], ke = it[DLFP_W_KVEND];
  const int nsplits = it[DLFP_W_NSPLITS];
  // First packed row and first position of the sequence's new tokens.
  const int q0 = it[DLFP_W_QROW0] - t0, pos0 = it[DLFP_W_QPOS0] - t0;
  const int32_t* bt = a.block_table + (int64_t)s * a.max_blocks;

  const int r = wave * 32 + col;       // this lane's row within the tile
  const int tr = r / G, hh = r % G;    // token within the unit, head within the group
  const bool row_ok = tr < nt;
  const int lim = row_ok ? min(pos0 + t0 + tr + 1, ke) : 0;  // keys < lim are visible
  const int wave_tok0 = uniform((wave * 32) / G);
  const bool wave_active = wave_tok0 < nt;
  const int wave_lim_min = min(pos0 + t0 + wave_tok0 + 1, ke);

  // Q^T as the B operand: lane holds dims [16kk + 8hi, +8) of its row.
  // Rows past the unit's tokens load the first row's query; they are never stored.
  bf16x8_t qf[8];
  {
    const int64_t qrow = ((int64_t)(q0 + t0 + (row_ok ? tr : 0)) * a.hq + kh * G + hh) * D;
#pragma unroll
    for (int kk = 0; kk < 8; ++kk)
      qf[kk] = *reinterpret_cast<const bf16x8_t*>(a.q + qrow + 16 * kk + 8 * hi);
  }

  const int ntiles = (ke - kb + KV_TILE - 1) / KV_TILE;
  const int first_page = kb / PAGE, last_page = (ke - 1) / PAGE;
  // Append launches: the first tile with a page at or past the one holding
  // the sequence's first new token (the unit waits before loading it).
  int wait_tile = ntiles;
  if constexpr (APP) {
    const int newp = pos0 / PAGE;
    if (a.app_wgs > 0 && last_page >= newp)
      wait_tile = max(0, (newp - first_page) >> 2);  // wave 3's page
  }
  int32_t* ptab = reinterpret_cast<int32_t*>(smem + PTAB_BASE);
  for (int i = tid; i <= last_page - first_page; i += THREADS) ptab[i] = bt[first_page + i];
  wait_memory_complete();  // queries and block ids resident before the KV pipeline starts
  __syncthreads();

  // Copies: wave w moves page w of each 64-key tile, its 16 K rows and its
  // 128 V^T rows, as four 1 KiB pieces each.  K row R keeps 16-byte chunk x
  // at position x ^ (R & 15); V^T row d keeps half h at position h ^ vt_swz(d).
  uint32_t koff[4], voff[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int rr = 4 * i + (lane >> 4);
    koff[i] = rr * 256 + (((lane & 15) ^ rr) << 4);
    const int d = 32 * i + (lane >> 1);
    voff[i] = d * 32 + (((lane & 1) ^ vt_swz(d)) << 4);
  }
  // Straight-line on purpose: a page past the unit's last key re-reads its
  // last page (every key there is masked), and a block id outside the pool is
  // replaced by block 0 after raising the error word.
  // Element offset of this wave's page of tile t (same in both caches).
  auto page_off = [&](int t) -> int64_t {
    const int page = min(first_page + 4 * t + wave, last_page);
    const int raw = uniform(ptab[page - first_page]);
    const bool ok = (unsigned)raw < (unsigned)a.num_blocks;
    if (!ok && lane == 0) raise_error(a.ws);
    return ((int64_t)(ok ? raw : 0) * a.hkv + kh) * PAGE_ELEMS;
  };
  const uint32_t lds_wave = lds_addr(smem) + uniform(wave) * (PAGE * 256);
  auto issue_k = [&](int64_t off, int slot) {
    const char* src = reinterpret_cast<const char*>(a.kc + off);
#pragma unroll
    for (int i = 0; i < 4; ++i) lds_copy16(src + koff[i], lds_wave + slot * TILE_BYTES + i * 1024);
  };
  auto issue_v = [&](int64_t off, int slot) {
    const char* src = reinterpret_cast<const char*>(a.vc + off);
#pragma unroll
    for (int i = 0; i < 4; ++i)
      lds_copy16(src + voff[i], lds_wave + V_BASE + slot * TILE_BYTES + i * 1024);
  };
  // Values past the unit's last key are zeroed in LDS (a probability of 0
  // times a NaN left in an unused slot would still be NaN).
  auto zero_v_tail = [&](int slot, int k0) {
    const int pg = tid >> 6;
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int d = 2 * (tid & 63) + (c >> 1), h = c & 1;
      char* p = smem + V_BASE + slot * TILE_BYTES + pg * (PAGE * 256) + d * 32 + (h << 4);
      const int half = h ^ vt_swz(d);
      const int key0 = k0 + pg * PAGE;
      *reinterpret_cast<u32x4_t*>(p) = mask_elems(*reinterpret_cast<const u32x4_t*>(p), ke,
                                                   [&](int e) { return key0 + vt_pos(8 * half + e); });
    }
  };

  // Per-lane LDS offsets.  K: chunk (2kk + hi) of row R = 32 kb2 + col sits at
  // ((2kk + hi) ^ (col & 15)) << 4, i.e. kbase ^ (kk << 5).  V^T: half hi of
  // dim row d = 32 mb + col, at a lane-constant offset plus immediates.
  const int kbase = col * 256 + ((hi ^ (col & 15)) << 4);
  const int vbase = V_BASE + col * 32 + ((hi ^ vt_swz(col)) << 4);

  float m_run = NEG_BIG, l_run = 0.f;
  f32x16_t o[4];
#pragma unroll
  for (int mb = 0; mb < 4; ++mb) o[mb] = f32x16_t{};
  const float c = a.scale_log2;

  // S^T = K Q^T for the 64 keys of the tile in K slot `slot`: two 32-key
  // accumulators advanced alternately.  sacc[kb2][rr] holds key
  // 32 kb2 + 8 (rr / 4) + 4 hi + rr % 4 of this lane's row.
  auto qk = [&](f32x16_t* sacc, int slot) {
    sacc[0] = f32x16_t{};
    sacc[1] = f32x16_t{};
#pragma unroll
    for (int kk = 0; kk < 8; ++kk) {
      const char* kp = smem + slot * TILE_BYTES + (kbase ^ (kk << 5));
      const bf16x8_t k0f = *reinterpret_cast<const bf16x8_t*>(kp);
      const bf16x8_t k1f = *reinterpret_cast<const bf16x8_t*>(kp + 32 * 256);
      sacc[0] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(k0f, qf[kk], sacc[0], 0, 0, 0);
      sacc[1] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(k1f, qf[kk], sacc[1], 0, 0, 0);
    }
  };
  // Causal and tail mask for a tile starting at key k0 (raw scores).
  auto mask = [&](f32x16_t* sacc, int k0) {
#pragma unroll
    for (int kb2 = 0; kb2 < 2; ++kb2)
#pragma unroll
      for (int rr = 0; rr < 16; ++rr) {
        const int key = k0 + kb2 * 32 + 8 * (rr >> 2) + 4 * hi + (rr & 3);
        sacc[kb2][rr] = key < lim ? sacc[kb2][rr] : -__builtin_inff();
      }
  };
  // Row maximum of a tile (raw scores), both halves of the row.
  auto rowmax = [&](const f32x16_t* sacc) {
    float mx = -__builtin_inff();
#pragma unroll
    for (int kb2 = 0; kb2 < 2; ++kb2)
#pragma unroll
      for (int rr = 0; rr < 16; ++rr) mx = fmaxf(mx, sacc[kb2][rr]);
    return max_xor32(mx);
  };
  // Raise the reference maximum where a tile exceeds it by more than
  // RESCALE_LOG2 (scaled units); the accumulators follow.
  auto rebase = [&](float mx) {
    const float m_tile = mx * c;
    if (__builtin_amdgcn_ballot_w64(m_tile > m_run + RESCALE_LOG2)) {
      const float m_new = m_tile > m_run + RESCALE_LOG2 ? m_tile : m_run;
      const float alpha = fexp2(m_run - m_new);
      m_run = m_new;
      l_run *= alpha;
#pragma unroll
      for (int mb = 0; mb < 4; ++mb) o[mb] *= alpha;
    }
  };
  // P^T = exp2(S^T c - m) rounded to bf16, as the B operands of the four
  // 16-key steps of PV; pf[kk] holds keys 16 kk + {0-3, 8-11} + 4 hi.
  auto probs = [&](const f32x16_t* sacc, bf16x8_t* pf) {
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      u32x4_t pk;
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        const float p0 = fexp2(__builtin_fmaf(sacc[kk >> 1][8 * (kk & 1) + 2 * w], c, -m_run));
        const float p1 = fexp2(__builtin_fmaf(sacc[kk >> 1][8 * (kk & 1) + 2 * w + 1], c, -m_run));
        pk[w] = pack_bf16(p0, p1);
      }
      pf[kk] = __builtin_bit_cast(bf16x8_t, pk);
    }
  };
  // Row sum of the rounded probabilities (this half of the row).
  auto rowsum = [&](const bf16x8_t* pf) {
    constexpr uint32_t ONES = 0x3F803F80u;  // two bf16 1.0
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      const u32x4_t pk = __builtin_bit_cast(u32x4_t, pf[kk]);
#pragma unroll
      for (int w = 0; w < 4; ++w) l_run = dot2(pk[w], ONES, l_run);
    }
  };
  // O^T += V^T P^T over the tile in V slot `slot`.
  auto pv = [&](const bf16x8_t* pf, int slot) {
#pragma unroll
    for (int kk = 0; kk < 4; ++kk)
#pragma unroll
      for (int mb = 0; mb < 4; ++mb) {
        const bf16x8_t vf = *reinterpret_cast<const bf16x8_t*>(
            smem + vbase + slot * TILE_BYTES + kk * (PAGE * 256) + mb * 1024);
        o[mb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf[kk], o[mb], 0, 0, 0);
      }
  };
  const bool tail = kb + ntiles * KV_TILE > ke;  // the last tile reaches past the unit's keys

  // Prologue: tiles 0 (K and V) and 1 (K) in flight, then S_0.  off_next
  // carries the page of tile j + 1 from the step that loaded its keys to the
  // step that loads its values.
  // The wait for the append records sits outside the tile loop (which is
  // split there): inside it, the poll's control flow costs the loop body its
  // partial LDS waits.  Tile t's keys are issued in the prologue (t < 2) or
  // by step t - 2.
  if constexpr (APP) {
    if (wait_tile <= 1) wait_for_appends(a);
  }
  int64_t off_next = page_off(0);
  issue_k(off_next, 0);
  issue_v(off_next, 0);
  if (ntiles > 1) {
    off_next = page_off(1);
    issue_k(off_next, 1);
  }
  wait_memory_complete();
  __syncthreads();
  if (tail && ntiles == 1) {
    zero_v_tail(0, kb);
    __syncthreads();
  }
  f32x16_t sa[2], sb[2];
  if (wave_active) {
    qk(sa, 0);
    if (kb + KV_TILE > wave_lim_min) mask(sa, kb);
    rebase(rowmax(sa));
  }
  __syncthreads();  // K slot 0 is refilled below

  // Iteration j: loads of K_{j+2} and V_{j+1} go out; S_{j+1} = K_{j+1} Q^T
  // runs on the matrix cores while the probabilities of tile j are formed;
  // then O += V_j P_j runs while the row maxima of tile j + 1 are taken.
  auto step = [&](int j, f32x16_t* cur, f32x16_t* nxt, auto parity) {
    constexpr int PAR = decltype(parity)::value;  // j & 1
    const bool more = j + 1 < ntiles;
    if (more) issue_v(off_next, PAR ^ 1);
    if (j + 2 < ntiles) {
      off_next = page_off(j + 2);
      issue_k(off_next, PAR);
    }
    if (wave_active) {
      bf16x8_t pf[4];
      // On the last tile this reads a stale slot; the result is not used, and
      // keeping it unconditional lets the products overlap the exponentials.
      qk(nxt, PAR ^ 1);
      probs(cur, pf);
      // Beside decode workgroups a prefill wavefront has no second prefill
      // wavefront on its SIMD to overlap with, so in a mixed launch the key
      // operands of the QK products are read four products ahead, one per
      // product, and the exponentials fill the gaps between the products.
      // Beside prefill wavefronts the compiler's own order is faster
      // (measured: Qwen3-32B sweep 0.8% faster with this order in mixed
      // launches, prefill-only launches 0.6-1% slower with it).
      if constexpr (MIXED) {
        __builtin_amdgcn_sched_group_barrier(0x100, 4, 0);
#pragma unroll
        for (int i = 0; i < 16; ++i) {
          __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
          __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        }
      }
      // The PV products and row sums run at raised wave priority: the SIMD
      // arbiter then keeps feeding the matrix core of the wave that is past
      // its exponentials while the other waves of the CU finish theirs
      // (measured 4-7% more prefill throughput on long chunks).
      __builtin_amdgcn_s_setprio(1);
      pv(pf, PAR);
      rowsum(pf);
      // Issue order of the raised-priority phase (s_setprio ends a scheduling
      // region, so these groups order the PV(j) products, the LDS reads of
      // their value operands and the row sums only).
      __builtin_amdgcn_sched_group_barrier(0x100, 4, 0);
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x002, 6, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      }
#pragma unroll
      for (int i = 0; i < 16; ++i) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x002, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      }
      __builtin_amdgcn_s_setprio(0);
      if (more) {
        const int k1 = kb + (j + 1) * KV_TILE;
        if (k1 + KV_TILE > wave_lim_min) mask(nxt, k1);
        rebase(rowmax(nxt));
      }
    }
    wait_memory_complete();
    __syncthreads();
    if (tail && j + 2 == ntiles) {  // V of the last tile has landed
      zero_v_tail(PAR ^ 1, kb + (ntiles - 1) * KV_TILE);
      __syncthreads();
    }
  };
  const std::integral_constant<int, 0> even;
  const std::integral_constant<int, 1> odd;
  int j = 0;
  if constexpr (APP) {
    if (wait_tile > 1 && wait_tile < ntiles) {
      const int jw = wait_tile - 2;  // the step that issues tile wait_tile
      for (; j + 1 < jw; j += 2) {
        step(j, sa, sb, even);
        step(j + 1, sb, sa, odd);
      }
      if (j < jw) step(j++, sa, sb, even);
      wait_for_appends(a);
      if (j & 1) step(j++, sb, sa, odd);
    }
  }
  for (; j < ntiles; j += 2) {
    step(j, sa, sb, even);
    if (j + 1 < ntiles) step(j + 1, sb, sa, odd);
  }

  // A waiting unit counts itself past its wait; the count returns while the
  // results are stored, and the last such unit zeroes the append words.
  int waited = -1;
  if constexpr (APP) {
    if (wait_tile < ntiles && tid == 0)
      waited = __hip_atomic_fetch_add(header_word(a.ws, HDR_WAITED), 1, __ATOMIC_RELAXED,
                                      __HIP_MEMORY_SCOPE_AGENT);
  }
  auto reset_append_words = [&]() {
    if constexpr (APP) {
      if (waited >= 0 && waited == a.num_waiting - 1) {
        __hip_atomic_store(header_word(a.ws, HDR_APPEND), 0, __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
        __hip_atomic_store(header_word(a.ws, HDR_WAITED), 0, __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
      }
    }
  };

  l_run = sum_xor32(l_run);
  const int rows = nt * G;
  // o[mb][rr] = O[row][32 mb + 8 (rr / 4) + 4 hi + rr % 4]
  if (nsplits == 1) {
    if (row_ok) {
      const float inv = 1.f / l_run;
      const int64_t orow = ((int64_t)(q0 + t0 + tr) * a.hq + kh * G + hh) * D;
#pragma unroll
      for (int mb = 0; mb < 4; ++mb)
#pragma unroll
        for (int g4 = 0; g4 < 4; ++g4)
          store4(a, orow + mb * 32 + 8 * g4 + 4 * hi, o[mb][4 * g4] * inv,
                 o[mb][4 * g4 + 1] * inv, o[mb][4 * g4 + 2] * inv, o[mb][4 * g4 + 3] * inv);
    }
    reset_append_words();
    return;
  }

  // Partial result: O as 16 chunks c = 4 mb + g4 of [rows][2][4] floats (chunk
  // c, row r, half h holds dims 32 mb + 8 g4 + 4 h .. + 3), so that a wave's
  // store and the merge's loads each cover a contiguous kilobyte; then
  // m[rows] and l[rows].
  const int slot_floats = slot_floats_for(rows);
  const Slots sl = group_slots(a.ws, it[DLFP_W_WSGROUP], nsplits, slot_floats);
  const int my = it[DLFP_W_SPLIT] * slot_floats;
  if (row_ok) {
#pragma unroll
    for (int mb = 0; mb < 4; ++mb)
#pragma unroll
      for (int g4 = 0; g4 < 4; ++g4) {
        const f32x4_t v = {o[mb][4 * g4], o[mb][4 * g4 + 1], o[mb][4 * g4 + 2],
                           o[mb][4 * g4 + 3]};
        pstore4(sl, my + ((4 * mb + g4) * rows + r) * 8 + 4 * hi, v);
      }
    if (hi == 0) {
      pstore1(sl, my + rows * D + r, m_run);
      pstore1(sl, my + rows * D + rows + r, l_run);
    }
  }
  wait_memory_complete();
  reset_append_words();
  __syncthreads();  // every wave of the unit has completed its stores
  const int grp = it[DLFP_W_GROUP];
  if (tid == 0) *flag = arrive(a.ws, grp) == nsplits - 1;
  __syncthreads();
  if (!*flag) return;

  // Last arriver: merge every split of the group (threads per row chosen so
  // that the whole workgroup takes part).
  if (rows > 64)
    prefill_merge<G, 2>(a, sl, slot_floats, nsplits, rows, q0 + t0, kh);
  else if (rows > 32)
    prefill_merge<G, 4>(a, sl, slot_floats, nsplits, rows, q0 + t0, kh);
  else
    prefill_merge<G, 8>(a, sl, slot_floats, nsplits, rows, q0 + t0, kh);
  if (tid == 0)
    __hip_atomic_store(group_counter(a.ws, grp), 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Last arriver of a decode split group: merges the group's partial results
// (O[G][128], m[G], l[G] per split, in split order) into the output.  Lane
// `lane` writes dims 2 lane and 2 lane + 1 of every head; obase is the
// element offset of those dims of the group's first head.
template <int G>
__device__ __forceinline__ void decode_merge(const Args& a, const Slots sl, int slot_floats,
                                             int nsplits, int64_t obase, int grp) {
  const int lane = threadIdx.x & 63;
  // Entry f = j G + h stands for head h of split j.  Per batch
  // of up to 64 entries, lane e loads entry e's maximum and row sum while
  // every lane loads its two dims of the batch's entries (in groups of 16,
  // only as many groups as the batch has entries), so a batch costs one
  // memory round trip; the running per-head maximum rescales what earlier
  // batches summed, and entries are accumulated in split order.
  const int nf = nsplits * G;
  float M[G], lsum[G], acc0[G], acc1[G];
#pragma unroll
  for (int h = 0; h < G; ++h) {
    M[h] = NEG_BIG;
    lsum[h] = acc0[h] = acc1[h] = 0.f;
  }
  for (int f0 = 0; f0 < nf; f0 += 64) {
    const int n = min(64, nf - f0);
    const int fl = f0 + min(lane, n - 1);
    const int lbase = (fl / G) * slot_floats + G * D + fl % G;
    const float mf = lane < n ? pload1(sl, lbase) : NEG_BIG;
    const float lf = pload1(sl, lbase + G);
    f32x2_t v[4][16];
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      if (16 * q < n) {
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int fe = f0 + min(16 * q + e, n - 1);
          v[q][e] = pload2(sl, (fe / G) * slot_floats + (fe % G) * D + 2 * lane);
        }
      }
    }
    // Batch maximum of head lane % G (f0 is a multiple of 64, so entry
    // f0 + e belongs to head e % G).
    float bm = mf;
#pragma unroll
    for (int sh = G; sh < 64; sh <<= 1) bm = fmaxf(bm, shfl_xor(bm, sh));
    float mh = NEG_BIG;
#pragma unroll
    for (int h = 0; h < G; ++h) {
      const float mnew = fmaxf(M[h], __builtin_bit_cast(float, __builtin_amdgcn_readlane(
                                                                  __builtin_bit_cast(int, bm), h)));
      const float rs = fexp2(M[h] - mnew);
      M[h] = mnew;
      lsum[h] *= rs;
      acc0[h] *= rs;
      acc1[h] *= rs;
      if (lane % G == h) mh = mnew;
    }
    const float wf = lane < n ? fexp2(mf - mh) : 0.f;
    const float wl = wf * lf;
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      if (16 * q < n) {
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int src = 16 * q + e;  // weights of entries past the batch are zero
          const float w = __builtin_bit_cast(float, __builtin_amdgcn_readlane(
                                                        __builtin_bit_cast(int, wf), src));
          const float lw = __builtin_bit_cast(float, __builtin_amdgcn_readlane(
                                                         __builtin_bit_cast(int, wl), src));
          lsum[e % G] += lw;
          acc0[e % G] += w * v[q][e][0];
          acc1[e % G] += w * v[q][e][1];
        }
      }
    }
  }
#pragma unroll
  for (int h = 0; h < G; ++h) {
    const float inv = 1.f / lsum[h];
    store2(a, obase + h * D, acc0[h] * inv, acc1[h] * inv);
  }
  if (lane == 0)
    __hip_atomic_store(group_counter(a.ws, grp), 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// ---------------------------------------------------------------- decode

// Wave-private LDS slice: two page slots, each a K page (token rows, 16-byte
// chunk x of row R at x ^ 8 (R & 1)) and a V^T page (64-byte dim-pair region
// r, 16-byte slot i at (i + r / 4) & 3); then the probability buffer
// p[head][16 keys] in bf16, the unit's block ids and (g = 8) the queries.
// Returns the next queue ticket's pending value when asked to take one (see
// the kernel's decode loop): the ticket is taken a few pages before the unit
// ends, so that its round trip overlaps the unit's last pages.
template <int G, bool APP>
__device__ int decode_unit(const Args& a, const int32_t* it_g, char* wl, bool take_ticket) {
  const int lane = threadIdx.x & 63;
  const int kg = lane >> 3, c = lane & 7;
  const record_ptr it = as_record(it_g);
  const int s = it[DLFP_W_SEQ], kh = it[DLFP_W_KVHEAD];
  const int kb = it[DLFP_W_KVBEGIN], ke = it[DLFP_W_KVEND];
  const int nsplits = it[DLFP_W_NSPLITS];
  const int tok = it[DLFP_W_QROW0];
  const int newpos = it[DLFP_W_QPOS0];
  const int first_blk = it[DLFP_W_PAGE0], second_blk = it[DLFP_W_PAGE1];
  const int grp = it[DLFP_W_GROUP], wsgroup = it[DLFP_W_WSGROUP], split = it[DLFP_W_SPLIT];
  const int32_t* bt = a.block_table + (int64_t)s * a.max_blocks;
  uint16_t* pbuf = reinterpret_cast<uint16_t*>(wl + 2 * DEC_PAGE_SLOT);
  int32_t* ptab = reinterpret_cast<int32_t*>(wl + 2 * DEC_PAGE_SLOT + 16 * 16 * 2);

  // Page pipeline.  Pages reach the slot's LDS by direct global-to-LDS copies
  // (no registers, no staging writes); each lane's source chunk is chosen so
  // that the bytes land in the swizzled layout above.  Without a prefill share
  // in the launch, page p + 2 is issued as soon as page p has been consumed,
  // so one to two pages (8-16 KiB) per wavefront stay in flight (HBM delivers
  // 6.0 TB/s to 8 wavefronts per CU with 8-16 KiB each in flight in a probe,
  // 5.3 TB/s with 4 KiB).  Beside a prefill share, page p + 1 is issued when
  // page p has landed, one page ahead: a deeper queue makes the prefill tiles
  // wait longer for their loads (measured 3.6-5.5% longer iterations for
  // chunks of 64-256 tokens).  A block id outside the pool is replaced by
  // block 0 after raising the error word.
  const bool deep = a.deep != 0;
  const int p_begin = kb / PAGE, p_end = (ke + PAGE - 1) / PAGE;
  const int npages = p_end - p_begin;
  uint32_t kofs[4], vofs[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int ck = 64 * j + lane;  // LDS chunk this lane fills
    const int R = ck >> 4, xs = ck & 15;
    kofs[j] = R * 256 + ((xs ^ ((R & 1) << 3)) << 4);
    const int rg = ck >> 2, si = ((ck & 3) - (rg >> 2)) & 3;
    vofs[j] = (rg * 4 + si) * 16;
  }
  const uint32_t lds_wave = (uint32_t)uniform((int)lds_addr(wl));
  auto issue_block = [&](int raw, int slot) {
    const bool ok = (unsigned)raw < (unsigned)a.num_blocks;
    if (!ok && lane == 0) raise_error(a.ws);
    const int64_t base = ((int64_t)(ok ? raw : 0) * a.hkv + kh) * PAGE_ELEMS;
    const char* ksrc = reinterpret_cast<const char*>(a.kc + base);
    const char* vsrc = reinterpret_cast<const char*>(a.vc + base);
    const uint32_t dst = lds_wave + uniform(slot) * DEC_PAGE_SLOT;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      lds_copy16_nt(ksrc + kofs[j], dst + j * 1024);
      lds_copy16_nt(vsrc + vofs[j], dst + PAGE_ELEMS * 2 + j * 1024);
    }
  };
  auto issue = [&](int p, int slot) { issue_block(uniform(ptab[p - p_begin]), slot); };
  // Vector-memory operations complete in issue order, so allowing the 8
  // copies of the next page to stay outstanding waits for this one.
  auto wait_page = [&](bool next_in_flight) {
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    if (next_in_flight)
      __builtin_amdgcn_s_waitcnt(0x0F78);  // vmcnt(8)
    else
      __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0)
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
  };

  // Prologue, one memory round trip after the work record: the first page
  // (its block id comes with the record), the queries, the unit's block ids
  // and (append launches) the new token's key and values all go out together,
  // then the second page when two are kept in flight.  Queries of g <= 4 heads
  // stay in registers (lane uses dims [8c, 8c + 8) and [64 + 8c, 64 + 8c + 8));
  // for g = 8 they go to the wave's LDS slice (each read is an 8-address
  // broadcast).  The append launch's unit whose keys end with the sequence's
  // new token (position QPOS0) loads that token's key row (lanes 0-15, 16
  // bytes each) and its values of dims 2 lane, 2 lane + 1, writes them to
  // their slot, and puts them into the landed page in place of what the cache
  // held there.
  issue_block(first_blk, 0);
  constexpr bool Q_IN_LDS = G >= 8;
  constexpr int QR = Q_IN_LDS ? 1 : G;
  u32x4_t qa[QR], qb[QR];
  uint16_t* qlds =
      reinterpret_cast<uint16_t*>(wl + 2 * DEC_PAGE_SLOT + 16 * 16 * 2 + DEC_PTAB * 4);
  const uint16_t* qp = a.q + ((int64_t)tok * a.hq + kh * G) * D;
  constexpr int QCH = Q_IN_LDS ? G * D / 8 / 64 : 1;  // 16-byte query chunks per lane (g = 8)
  u32x4_t qv[QCH];
  if constexpr (Q_IN_LDS) {
#pragma unroll
    for (int k = 0; k < QCH; ++k)
      qv[k] = *reinterpret_cast<const u32x4_t*>(qp + 8 * (lane + 64 * k));
  } else {
#pragma unroll
    for (int h = 0; h < G; ++h) {
      qa[h] = *reinterpret_cast<const u32x4_t*>(qp + h * D + 8 * c);
      qb[h] = *reinterpret_cast<const u32x4_t*>(qp + h * D + 64 + 8 * c);
    }
  }
  constexpr int PTV = DEC_PTAB / 64;
  int ptv[PTV];
#pragma unroll
  for (int k = 0; k < PTV; ++k) {
    const int i = lane + 64 * k;
    ptv[k] = i < npages ? bt[p_begin + i] : 0;
  }
  const bool own_new = APP && newpos < ke;
  const int new_page = newpos / PAGE, new_off = newpos % PAGE;
  u32x4_t kn = {0u, 0u, 0u, 0u};
  uint32_t vn = 0u;
  if (own_new) {
    const int64_t src = ((int64_t)tok * a.hkv + kh) * D;
    if (lane < 16) kn = *reinterpret_cast<const u32x4_t*>(a.k_new + src + 8 * lane);
    vn = *reinterpret_cast<const uint32_t*>(a.v_new + src + 2 * lane);
  }
  if (deep && npages > 1) issue_block(second_blk, 1);
  wait_memory_complete();  // everything above has landed
  if constexpr (Q_IN_LDS) {
#pragma unroll
    for (int k = 0; k < QCH; ++k) *reinterpret_cast<u32x4_t*>(qlds + 8 * (lane + 64 * k)) = qv[k];
  }
#pragma unroll
  for (int k = 0; k < PTV; ++k)
    if (lane + 64 * k < npages) ptab[lane + 64 * k] = ptv[k];
  wave_sync();
  if (own_new) {
    const int raw = ptab[new_page - p_begin];
    if ((unsigned)raw < (unsigned)a.num_blocks) {
      const int64_t base = ((int64_t)raw * a.hkv + kh) * PAGE_ELEMS;
      uint16_t* kc = const_cast<uint16_t*>(a.kc);
      uint16_t* vc = const_cast<uint16_t*>(a.vc);
      if (lane < 16) *reinterpret_cast<u32x4_t*>(kc + base + new_off * D + 8 * lane) = kn;
      vc[base + (2 * lane) * PAGE + vt_pos(new_off)] = (uint16_t)(vn & 0xFFFFu);
      vc[base + (2 * lane + 1) * PAGE + vt_pos(new_off)] = (uint16_t)(vn >> 16);
    }
  }
  float m[G], l[G], o0[G], o1[G];
#pragma unroll
  for (int h = 0; h < G; ++h) {
    m[h] = NEG_BIG;
    l[h] = 0.f;
    o0[h] = 0.f;
    o1[h] = 0.f;
  }
  // Queue mode: the next ticket is taken a few pages before the unit ends.
  int ticket_v = 0;
  const int ticket_page = max(p_begin, p_end - 4);

  auto process = [&](int p, int slot) {
    char* kl = wl + slot * DEC_PAGE_SLOT;
    char* vl = kl + PAGE_ELEMS * 2;
    wait_page(deep && p + 1 < p_end);
    wave_sync();
    if (!deep && p + 1 < p_end) issue(p + 1, slot ^ 1);  // that slot was consumed
    if (take_ticket && p == ticket_page && lane == 0)
      ticket_v = __hip_atomic_fetch_add(header_word(a.ws, HDR_TICKET), 1, __ATOMIC_RELAXED,
                                        __HIP_MEMORY_SCOPE_AGENT);
    if (p * PAGE + PAGE > ke) {
      // Values past the unit's last key are zeroed (a probability of 0 times
      // a NaN left in an unused slot would still be NaN).
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int ck = 64 * j + lane;
        const int rg = ck >> 2, si = ((ck & 3) - (rg >> 2)) & 3;
        u32x4_t* v = reinterpret_cast<u32x4_t*>(vl + ck * 16);
        *v = mask_elems(*v, ke, [&](int e) { return p * PAGE + vt_pos(8 * (si & 1) + e); });
      }
    }
    if (own_new && p == new_page) {
      if (lane < 16)
        *reinterpret_cast<u32x4_t*>(kl + new_off * 256 + ((lane ^ ((new_off & 1) << 3)) << 4)) = kn;
      // region lane holds dim 2 lane in slots 0-1 and dim 2 lane + 1 in slots 2-3
      const int sp = vt_pos(new_off), half = sp >> 3;
      char* v0 = vl + lane * 64 + (((half + (lane >> 2)) & 3) << 4) + 2 * (sp & 7);
      char* v1 = vl + lane * 64 + (((2 + half + (lane >> 2)) & 3) << 4) + 2 * (sp & 7);
      *reinterpret_cast<uint16_t*>(v0) = (uint16_t)(vn & 0xFFFFu);
      *reinterpret_cast<uint16_t*>(v1) = (uint16_t)(vn >> 16);
    }
    wave_sync();  // fixed-up page visible to every lane

    // Keys 8 st + kg of the page (st = 0, 1): each lane holds 16 dims of both.
    u32x4_t kv[2][2];
#pragma unroll
    for (int st = 0; st < 2; ++st) {
      const int R = 8 * st + kg;
      kv[st][0] = *reinterpret_cast<const u32x4_t*>(kl + R * 256 + ((c ^ ((R & 1) << 3)) << 4));
      kv[st][1] =
          *reinterpret_cast<const u32x4_t*>(kl + R * 256 + (((c + 8) ^ ((R & 1) << 3)) << 4));
    }
    const bool valid0 = p * PAGE + kg < ke, valid1 = p * PAGE + 8 + kg < ke;
    // One head at a time: scores (dot products summed over the 8 lanes of a
    // key), online-softmax update, probabilities to LDS, accumulator rescale.
#pragma unroll
    for (int h = 0; h < G; ++h) {
      u32x4_t qah, qbh;
      if constexpr (Q_IN_LDS) {
        qah = *reinterpret_cast<const u32x4_t*>(qlds + h * D + 8 * c);
        qbh = *reinterpret_cast<const u32x4_t*>(qlds + h * D + 64 + 8 * c);
      } else {
        qah = qa[h];
        qbh = qb[h];
      }
      float sc[2];
#pragma unroll
      for (int st = 0; st < 2; ++st) {
        float acc = 0.f;
#pragma unroll
        for (int w = 0; w < 4; ++w) acc = dot2(qah[w], kv[st][0][w], acc);
#pragma unroll
        for (int w = 0; w < 4; ++w) acc = dot2(qbh[w], kv[st][1][w], acc);
        acc += dpp<DPP_XOR1>(acc);
        acc += dpp<DPP_XOR2>(acc);
        acc += dpp<DPP_HALF_MIRROR>(acc);
        sc[st] = acc * a.scale_log2;
      }
      sc[0] = valid0 ? sc[0] : -__builtin_inff();
      sc[1] = valid1 ? sc[1] : -__builtin_inff();
      float mx = fmaxf(sc[0], sc[1]);
      mx = fmaxf(mx, dpp<DPP_ROR8>(mx));
      mx = max_xor16(mx);
      mx = max_xor32(mx);
      const float m_new = fmaxf(m[h], mx);
      const float alpha = fexp2(m[h] - m_new);
      m[h] = m_new;
      const float p0 = fexp2(sc[0] - m_new), p1 = fexp2(sc[1] - m_new);
      l[h] = l[h] * alpha + (c == 0 ? p0 + p1 : 0.f);
      o0[h] *= alpha;
      o1[h] *= alpha;
      if (c == (h & 7)) {
        pbuf[h * 16 + vt_pos(kg)] = __builtin_bit_cast(uint16_t, (__bf16)p0);
        pbuf[h * 16 + vt_pos(8 + kg)] = __builtin_bit_cast(uint16_t, (__bf16)p1);
      }
      if constexpr (G >= 8) __builtin_amdgcn_sched_barrier(0);  // bound live ranges per head
    }
    wave_sync();  // probabilities visible to every lane
    // O += P V: lane owns dims 2 lane and 2 lane + 1.
    u32x4_t vr[4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
      vr[i] = *reinterpret_cast<const u32x4_t*>(vl + lane * 64 + (((i + (lane >> 2)) & 3) << 4));
#pragma unroll
    for (int h = 0; h < G; ++h) {
      const u32x4_t pp0 = *reinterpret_cast<const u32x4_t*>(pbuf + h * 16);
      const u32x4_t pp1 = *reinterpret_cast<const u32x4_t*>(pbuf + h * 16 + 8);
      float a0 = o0[h], a1 = o1[h];
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        a0 = dot2(pp0[w], vr[0][w], a0);
        a1 = dot2(pp0[w], vr[2][w], a1);
      }
#pragma unroll
      for (int w = 0; w < 4; ++w) {
        a0 = dot2(pp1[w], vr[1][w], a0);
        a1 = dot2(pp1[w], vr[3][w], a1);
      }
      o0[h] = a0;
      o1[h] = a1;
      if constexpr (G >= 8) __builtin_amdgcn_sched_barrier(0);
    }
    wave_sync();  // every lane done reading the slot before it is refilled
    if (deep && p + 2 < p_end) issue(p + 2, slot);
  };

  for (int p = p_begin; p < p_end; p += 2) {
    process(p, 0);
    if (p + 1 < p_end) process(p + 1, 1);
  }

  // Row sums live on the c == 0 lanes; total them.
#pragma unroll
  for (int h = 0; h < G; ++h) {
    float x = l[h];
    x += dpp<DPP_ROR8>(x);
    x = sum_xor16(x);
    x = sum_xor32(x);
    l[h] = __builtin_bit_cast(float, uniform(__builtin_bit_cast(int, x)));
  }

  const int64_t obase = ((int64_t)tok * a.hq + kh * G) * D + 2 * lane;
  if (nsplits == 1) {
#pragma unroll
    for (int h = 0; h < G; ++h) {
      const float inv = 1.f / l[h];
      store2(a, obase + h * D, o0[h] * inv, o1[h] * inv);
    }
    return ticket_v;
  }

  // Partial: O[G][128], m[G], l[G].
  const int slot_floats = slot_floats_for(G);
  const Slots sl = group_slots(a.ws, wsgroup, nsplits, slot_floats);
  const int my = split * slot_floats;
#pragma unroll
  for (int h = 0; h < G; ++h) {
    pstore2(sl, my + h * D + 2 * lane, f32x2_t{o0[h], o1[h]});
    if (lane == 0) {
      pstore1(sl, my + G * D + h, m[h]);
      pstore1(sl, my + G * D + G + h, l[h]);
    }
  }
  wait_memory_complete();
  int old = 0;
  if (lane == 0) old = arrive(a.ws, grp);
  old = __shfl(old, 0);
  if (old != nsplits - 1) return ticket_v;

  decode_merge<G>(a, sl, slot_floats, nsplits, obase, grp);
  return ticket_v;
}

// ---------------------------------------------------------------- decode on the matrix cores

typedef short s16x4_t __attribute__((ext_vector_type(4)));

// Decode unit for g >= 2 query heads per KV head.  The unit's g heads are the
// columns of 16x16 matrix products (padded to 16 with zero queries): per page,
// the scores are S^T = K Q^T (four v_mfma_f32_16x16x32_bf16 over the 128
// dims) and the output advances by O^T += V^T P^T (eight
// v_mfma_f32_16x16x16_bf16 over the page's 16 keys), so the VALU only forms
// the softmax.  Lane l owns head column l % 16 and accumulator rows
// 4 (l / 16) .. + 3.  Row r of the K operand (and so of S^T) is token slot
// vt_pos(r) of the page: a lane's four rows are then four consecutive
// positions of a value-page row (the cache keeps V^T pages with slot t at
// position vt_pos(t)), so the probabilities go from the score accumulator
// straight into the B operand of the PV product, and a lane's V^T operand is
// one 8-byte LDS read.  Per-head maxima combine the four lane groups with
// permlane swaps; the reference maximum is raised lazily, as in the prefill
// tiles.
//
// LDS page slots (two per wavefront, as for decode_unit): K page row R keeps
// its 16-byte chunk x at position x ^ R; V^T row d (32 bytes) keeps its two
// 16-byte halves swapped when bit 3 of d is set.  Either way the lanes that
// LDS serves together read distinct banks.  The page pipeline, the prologue,
// the queue tickets, the one-launch append and the split merge are those of
// decode_unit.
template <int G, bool APP>
__device__ int decode_unit_mfma(const Args& a, const int32_t* it_g, char* wl, bool take_ticket) {
  static_assert(G >= 2 && G <= 16, "heads must fit the 16 columns");
  const int lane = threadIdx.x & 63;
  const int col = lane & 15, gq = lane >> 4;
  const record_ptr it = as_record(it_g);
  const int s = it[DLFP_W_SEQ], kh = it[DLFP_W_KVHEAD];
  const int kb = it[DLFP_W_KVBEGIN], ke = it[DLFP_W_KVEND];
  const int nsplits = it[DLFP_W_NSPLITS];
  const int tok = it[DLFP_W_QROW0];
  const int newpos = it[DLFP_W_QPOS0];
  const int first_blk = it[DLFP_W_PAGE0], second_blk = it[DLFP_W_PAGE1];
  const int grp = it[DLFP_W_GROUP], wsgroup = it[DLFP_W_WSGROUP], split = it[DLFP_W_SPLIT];
  const int32_t* bt = a.block_table + (int64_t)s * a.max_blocks;
  int32_t* ptab = reinterpret_cast<int32_t*>(wl + 2 * DEC_PAGE_SLOT + 16 * 16 * 2);

  const bool deep = a.deep != 0;
  const int p_begin = kb / PAGE, p_end = (ke + PAGE - 1) / PAGE;
  const int npages = p_end - p_begin;
  uint32_t kofs[4], vofs[4];
#pragma unroll
  for (int j = 0; j < 4; ++j) {
    const int ck = 64 * j + lane;  // LDS chunk this lane fills
    const int R = ck >> 4, xs = ck & 15;
    kofs[j] = R * 256 + ((xs ^ R) << 4);
    const int d = ck >> 1, hs = ck & 1;
    vofs[j] = d * 32 + ((hs ^ ((d >> 3) & 1)) << 4);
  }
  const uint32_t lds_wave = (uint32_t)uniform((int)lds_addr(wl));
  auto issue_block = [&](int raw, int slot) {
    const bool ok = (unsigned)raw < (unsigned)a.num_blocks;
    if (!ok && lane == 0) raise_error(a.ws);
    const int64_t base = ((int64_t)(ok ? raw : 0) * a.hkv + kh) * PAGE_ELEMS;
    const char* ksrc = reinterpret_cast<const char*>(a.kc + base);
    const char* vsrc = reinterpret_cast<const char*>(a.vc + base);
    const uint32_t dst = lds_wave + uniform(slot) * DEC_PAGE_SLOT;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      lds_copy16_nt(ksrc + kofs[j], dst + j * 1024);
      lds_copy16_nt(vsrc + vofs[j], dst + PAGE_ELEMS * 2 + j * 1024);
    }
  };
  auto issue = [&](int p, int slot) { issue_block(uniform(ptab[p - p_begin]), slot); };
  auto wait_page = [&](bool next_in_flight) {
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
    if (next_in_flight)
      __builtin_amdgcn_s_waitcnt(0x0F78);  // vmcnt(8)
    else
      __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0)
    __atomic_signal_fence(__ATOMIC_SEQ_CST);
  };

  // Prologue (one round trip after the work record): the first page, the
  // queries as the B operand (lane holds dims 32 kk + 8 (l / 16) .. + 8 of head
  // column l % 16, zero past the unit's g heads), the unit's block ids and
  // (append launches) the new token's key row and value pair.
  issue_block(first_blk, 0);
  bf16x8_t qb[4];
  {
    const uint16_t* qp = a.q + ((int64_t)tok * a.hq + kh * G + min(col, G - 1)) * D + 8 * gq;
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      const u32x4_t v = *reinterpret_cast<const u32x4_t*>(qp + 32 * kk);
      qb[kk] = __builtin_bit_cast(bf16x8_t, col < G ? v : u32x4_t{0u, 0u, 0u, 0u});
    }
  }
  constexpr int PTV = DEC_PTAB / 64;
  int ptv[PTV];
#pragma unroll
  for (int k = 0; k < PTV; ++k) {
    const int i = lane + 64 * k;
    ptv[k] = i < npages ? bt[p_begin + i] : 0;
  }
  const bool own_new = APP && newpos < ke;
  const int new_page = newpos / PAGE, new_off = newpos % PAGE;
  u32x4_t kn = {0u, 0u, 0u, 0u};
  uint32_t vn = 0u;
  if (own_new) {
    const int64_t src = ((int64_t)tok * a.hkv + kh) * D;
    if (lane < 16) kn = *reinterpret_cast<const u32x4_t*>(a.k_new + src + 8 * lane);
    vn = *reinterpret_cast<const uint32_t*>(a.v_new + src + 2 * lane);
  }
  if (deep && npages > 1) issue_block(second_blk, 1);
  wait_memory_complete();
#pragma unroll
  for (int k = 0; k < PTV; ++k)
    if (lane + 64 * k < npages) ptab[lane + 64 * k] = ptv[k];
  wave_sync();
  if (own_new) {
    const int raw = ptab[new_page - p_begin];
    if ((unsigned)raw < (unsigned)a.num_blocks) {
      const int64_t base = ((int64_t)raw * a.hkv + kh) * PAGE_ELEMS;
      uint16_t* kc = const_cast<uint16_t*>(a.kc);
      uint16_t* vc = const_cast<uint16_t*>(a.vc);
      if (lane < 16) *reinterpret_cast<u32x4_t*>(kc + base + new_off * D + 8 * lane) = kn;
      vc[base + (2 * lane) * PAGE + vt_pos(new_off)] = (uint16_t)(vn & 0xFFFFu);
      vc[base + (2 * lane + 1) * PAGE + vt_pos(new_off)] = (uint16_t)(vn >> 16);
    }
  }

  float m_run = NEG_BIG, l_run = 0.f;
  f32x4_t o[8];
#pragma unroll
  for (int mb = 0; mb < 8; ++mb) o[mb] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  const float c = a.scale_log2;
  int ticket_v = 0;
  const int ticket_page = max(p_begin, p_end - 4);
  // This lane's K operand row (token slot vt_pos(col)), the token slot of its
  // first accumulator row (vt_pos(4 gq)), and its V^T operand's byte offset
  // inside a 16-row block (row col, positions 4 gq .. + 3).
  const int ra = vt_pos(col);
  const int slot0 = vt_pos(4 * gq);
  const int vbyte = col * 32 + (((gq >> 1) ^ ((col >> 3) & 1)) << 4) + 8 * (gq & 1);

  auto process = [&](int p, int slot) {
    char* kl = wl + slot * DEC_PAGE_SLOT;
    char* vl = kl + PAGE_ELEMS * 2;
    wait_page(deep && p + 1 < p_end);
    wave_sync();
    if (!deep && p + 1 < p_end) issue(p + 1, slot ^ 1);  // that slot was consumed
    if (take_ticket && p == ticket_page && lane == 0)
      ticket_v = __hip_atomic_fetch_add(header_word(a.ws, HDR_TICKET), 1, __ATOMIC_RELAXED,
                                        __HIP_MEMORY_SCOPE_AGENT);
    if (p * PAGE + PAGE > ke) {
      // Values past the unit's last key are zeroed (a probability of 0 times
      // a NaN left in an unused slot would still be NaN).
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int ck = 64 * j + lane;
        const int d = ck >> 1, h = (ck & 1) ^ ((d >> 3) & 1);
        u32x4_t* v = reinterpret_cast<u32x4_t*>(vl + ck * 16);
        *v = mask_elems(*v, ke, [&](int e) { return p * PAGE + vt_pos(8 * h + e); });
      }
    }
    if (own_new && p == new_page) {
      if (lane < 16)
        *reinterpret_cast<u32x4_t*>(kl + new_off * 256 + ((lane ^ new_off) << 4)) = kn;
      const int sp = vt_pos(new_off), half = sp >> 3;
      const int d0 = 2 * lane, d1 = 2 * lane + 1;
      *reinterpret_cast<uint16_t*>(vl + d0 * 32 + ((half ^ ((d0 >> 3) & 1)) << 4) + 2 * (sp & 7)) =
          (uint16_t)(vn & 0xFFFFu);
      *reinterpret_cast<uint16_t*>(vl + d1 * 32 + ((half ^ ((d1 >> 3) & 1)) << 4) + 2 * (sp & 7)) =
          (uint16_t)(vn >> 16);
    }
    wave_sync();  // fixed-up page visible to every lane

    // S^T = K Q^T: rows = token slots vt_pos(r), columns = heads.
    f32x4_t sacc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      const bf16x8_t kf =
          *reinterpret_cast<const bf16x8_t*>(kl + ra * 256 + (((4 * kk + gq) ^ ra) << 4));
      sacc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf, qb[kk], sacc, 0, 0, 0);
    }
    // Rows 4 gq + i hold slots slot0 + i; keys at or past ke are masked.
    float sc[4];
    float mx = -__builtin_inff();
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      sc[i] = p * PAGE + slot0 + i < ke ? sacc[i] : -__builtin_inff();
      mx = fmaxf(mx, sc[i]);
    }
    mx = max_xor32(max_xor16(mx));
    const float m_tile = mx * c;
    if (__builtin_amdgcn_ballot_w64(m_tile > m_run + RESCALE_LOG2)) {
      const float m_new = m_tile > m_run + RESCALE_LOG2 ? m_tile : m_run;
      const float alpha = fexp2(m_run - m_new);
      m_run = m_new;
      l_run *= alpha;
#pragma unroll
      for (int mb = 0; mb < 8; ++mb) o[mb] *= alpha;
    }
    // P^T rounded to bf16: this lane's keys of its head column, the B operand.
    u32x2_t pk;
    pk[0] = pack_bf16(fexp2(__builtin_fmaf(sc[0], c, -m_run)),
                      fexp2(__builtin_fmaf(sc[1], c, -m_run)));
    pk[1] = pack_bf16(fexp2(__builtin_fmaf(sc[2], c, -m_run)),
                      fexp2(__builtin_fmaf(sc[3], c, -m_run)));
    constexpr uint32_t ONES = 0x3F803F80u;  // two bf16 1.0
    l_run = dot2(pk[1], ONES, dot2(pk[0], ONES, l_run));
    const s16x4_t pb = __builtin_bit_cast(s16x4_t, pk);
    // O^T += V^T P^T, eight blocks of 16 dims.
#pragma unroll
    for (int mb = 0; mb < 8; ++mb) {
      const s16x4_t vf = *reinterpret_cast<const s16x4_t*>(vl + mb * 512 + vbyte);
      o[mb] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(vf, pb, o[mb], 0, 0, 0);
    }
    wave_sync();  // every lane done reading the slot before it is refilled
    if (deep && p + 2 < p_end) issue(p + 2, slot);
  };

  for (int p = p_begin; p < p_end; p += 2) {
    process(p, 0);
    if (p + 1 < p_end) process(p + 1, 1);
  }

  // Row sums: each lane group holds a quarter of the keys of its head.
  const float l_tot = sum_xor32(sum_xor16(l_run));
  // o[mb][i] = O[head col][16 mb + 4 gq + i]
  if (nsplits == 1) {
    if (col < G) {
      const float inv = 1.f / l_tot;
      const int64_t orow = ((int64_t)tok * a.hq + kh * G + col) * D + 4 * gq;
#pragma unroll
      for (int mb = 0; mb < 8; ++mb)
        store4(a, orow + 16 * mb, o[mb][0] * inv, o[mb][1] * inv, o[mb][2] * inv,
               o[mb][3] * inv);
    }
    return ticket_v;
  }

  // Partial: O[G][128], m[G], l[G].
  const int slot_floats = slot_floats_for(G);
  const Slots sl = group_slots(a.ws, wsgroup, nsplits, slot_floats);
  const int my = split * slot_floats;
  if (col < G) {
#pragma unroll
    for (int mb = 0; mb < 8; ++mb) pstore4(sl, my + col * D + 16 * mb + 4 * gq, o[mb]);
    if (gq == 0) {
      pstore1(sl, my + G * D + col, m_run);
      pstore1(sl, my + G * D + G + col, l_tot);
    }
  }
  wait_memory_complete();
  int old = 0;
  if (lane == 0) old = arrive(a.ws, grp);
  old = __shfl(old, 0);
  if (old != nsplits - 1) return ticket_v;
  decode_merge<G>(a, sl, slot_floats, nsplits, ((int64_t)tok * a.hq + kh * G) * D + 2 * lane,
                  grp);
  return ticket_v;
}

// ---------------------------------------------------------------- append

// Append workgroup (append launches): each wavefront writes whole append
// records, one at a time -- one run of a prompt sequence's new tokens inside
// one page, for one KV head.  Key rows: lane covers 16-byte chunk lane % 16
// of rows 4 j + lane / 16.  Values: lane owns dims 2 lane and 2 lane + 1 and
// gathers them with one 4-byte load per token (a wavefront reads the whole
// 256-byte value row); a record that fills its page is written as whole
// 32-byte V^T rows, any other as one 2-byte value per token and dim (the
// page's other slots are left alone).  Every load of a record is issued
// before its stores.  The stores are ordinary ones, which the XCD's L2
// combines into whole lines (written through one by one, the half-line
// pieces cost a read-modify-write each at the memory side; measured 60-70 us
// for a 2048-token chunk).  When prefill units of the launch wait for the
// records, the workgroup then writes its L2 back (an agent-scope release) and
// counts itself done.

__device__ void append_records(const Args& a) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  uint16_t* kc = const_cast<uint16_t*>(a.kc);
  uint16_t* vc = const_cast<uint16_t*>(a.vc);
  const int x16 = lane & 15;
  for (int r = blockIdx.x * 4 + wave; r < a.num_append; r += 4 * a.app_wgs) {
    const int32_t* it = a.work + (int64_t)(a.num_units + r) * DLFP_WORK_INTS;
    const int s = uniform(it[DLFP_W_SEQ]), kh = uniform(it[DLFP_W_KVHEAD]);
    const int n = uniform(it[DLFP_W_QNTOK]), row0 = uniform(it[DLFP_W_QROW0]);
    const int pos = uniform(it[DLFP_W_QPOS0]);
    const int o0 = pos % PAGE, o1 = o0 + n;
    const int raw = uniform(a.block_table[(int64_t)s * a.max_blocks + pos / PAGE]);
    if ((unsigned)raw >= (unsigned)a.num_blocks || o1 > PAGE) {
      if (lane == 0) raise_error(a.ws);
      continue;
    }
    const int64_t base = ((int64_t)raw * a.hkv + kh) * PAGE_ELEMS;
    // token row of slot o in k_new / v_new: row0 + o - o0
    const int64_t src0 = ((int64_t)(row0 - o0) * a.hkv + kh) * D;
    const int64_t tok_stride = (int64_t)a.hkv * D;
    u32x4_t kr[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int o = 4 * j + (lane >> 4);
      kr[j] = o >= o0 && o < o1
                  ? *reinterpret_cast<const u32x4_t*>(a.k_new + src0 + o * tok_stride + 8 * x16)
                  : u32x4_t{0u, 0u, 0u, 0u};
    }
    uint32_t x[PAGE];
#pragma unroll
    for (int o = 0; o < PAGE; ++o)
      x[o] = o >= o0 && o < o1
                 ? *reinterpret_cast<const uint32_t*>(a.v_new + src0 + o * tok_stride + 2 * lane)
                 : 0u;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int o = 4 * j + (lane >> 4);
      if (o >= o0 && o < o1) *reinterpret_cast<u32x4_t*>(kc + base + o * D + 8 * x16) = kr[j];
    }
    uint16_t* row = vc + base + (2 * lane) * PAGE;  // rows 2 lane and 2 lane + 1
    if (o0 == 0 && o1 == PAGE) {
      // position 2 w + i of a row holds slot vt_pos(2 w + i)
      u32x4_t lo[2], hi[2];
#pragma unroll
      for (int w = 0; w < 8; ++w) {
        const uint32_t xa = x[vt_pos(2 * w)], xb = x[vt_pos(2 * w + 1)];
        lo[w >> 2][w & 3] = (xa & 0xFFFFu) | (xb << 16);
        hi[w >> 2][w & 3] = (xa >> 16) | (xb & 0xFFFF0000u);
      }
      u32x4_t* dst = reinterpret_cast<u32x4_t*>(row);
      dst[0] = lo[0];
      dst[1] = lo[1];
      dst[2] = hi[0];
      dst[3] = hi[1];
    } else {
#pragma unroll
      for (int o = 0; o < PAGE; ++o)
        if (o >= o0 && o < o1) {
          row[vt_pos(o)] = (uint16_t)(x[o] & 0xFFFFu);
          row[PAGE + vt_pos(o)] = (uint16_t)(x[o] >> 16);
        }
    }
  }
  if (a.num_waiting > 0) {
    wait_memory_complete();  // this wavefront's stores have reached the L2
    __syncthreads();
    if (threadIdx.x == 0) {
      __builtin_amdgcn_fence(__ATOMIC_RELEASE, "agent");  // write the L2 back
      __hip_atomic_fetch_add(header_word(a.ws, HDR_APPEND), 1, __ATOMIC_RELAXED,
                             __HIP_MEMORY_SCOPE_AGENT);
    }
  }
}

// The append records alone, as a launch of their own (one record per
// wavefront) ahead of the attention launch.
__global__ __launch_bounds__(THREADS) void append_records_kernel(Args a) { append_records(a); }

// ---------------------------------------------------------------- kernel

template <int G, bool APP, bool MIXED>
__global__ __launch_bounds__(THREADS, 2) void attention_mixed_kernel(Args a) {
  __shared__ __attribute__((aligned(16))) char smem[LDS_BYTES];
  __shared__ int flag;
  int b = blockIdx.x;
  if constexpr (APP) {
    // Append workgroups first (a multiple of 8, so the XCD of every later
    // workgroup is unchanged by the offset).
    if (b < a.app_wgs) {
      append_records(a);
      return;
    }
    b -= a.app_wgs;
  }
  // Grid: `lead` prefill workgroups, `decode_lead` decode workgroups, the
  // other prefill workgroups, the other decode workgroups.  The i-th prefill
  // workgroup takes unit xcd_remap(i): decode_lead is a multiple of 8, so the
  // i-th prefill workgroup runs on XCD i % 8 either way.
  const int np = a.num_prefill, L = a.lead, DL = a.decode_lead;
  int pi = -1, d = -1;
  if (b < L)
    pi = b;
  else if (b < L + DL)
    d = b - L;
  else if (b < np + DL)
    pi = b - DL;
  else
    d = b - np;
  if (pi >= 0) {
    const int u = xcd_remap(pi, np);
    prefill_unit<G, APP, MIXED>(a, a.work + (int64_t)u * DLFP_WORK_INTS, smem, &flag);
  } else {
    // Decode wavefront w of decode workgroup d starts with unit 4 d + w when
    // that is one of the first decode_static units (the workgroups resident
    // from the start); the other units form a queue that wavefronts drain one
    // ticket at a time as they finish, so none idles while units remain (a
    // workgroup's slot frees only when all four of its wavefronts are done),
    // and a workgroup that only becomes resident later takes tickets from the
    // start instead of holding units back to the tail.  The last workgroup to
    // finish resets the header words for the next launch.
    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    char* wl = smem + wave * DEC_WAVE_LDS;
    const int ndec = a.num_units - a.num_prefill;
    const bool queue = ndec > a.decode_static;
    auto ticket = [&]() {
      int nt = 0;
      if (lane == 0)
        nt = a.decode_static + __hip_atomic_fetch_add(header_word(a.ws, HDR_TICKET), 1,
                                                      __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      return uniform(__shfl(nt, 0));
    };
    int t = d * 4 + wave;
    if (queue && t >= a.decode_static) t = ticket();
    while (t < ndec) {
      // In queue mode the unit takes the next ticket itself near its end.
      const int32_t* rec = a.work + (int64_t)(a.num_prefill + t) * DLFP_WORK_INTS;
      int pending;
      if constexpr (G >= 2)
        pending = decode_unit_mfma<G, APP>(a, rec, wl, queue);
      else
        pending = decode_unit<G, APP>(a, rec, wl, queue);
      wave_sync();
      if (!queue) break;
      t = a.decode_static + uniform(__shfl(pending, 0));
    }
    if (queue) {
      __syncthreads();
      if (threadIdx.x == 0) {
        const int d = __hip_atomic_fetch_add(header_word(a.ws, HDR_DONE), 1, __ATOMIC_RELAXED,
                                             __HIP_MEMORY_SCOPE_AGENT);
        if (d == a.decode_waves / 4 - 1) {
          __hip_atomic_store(header_word(a.ws, HDR_TICKET), 0, __ATOMIC_RELAXED,
                             __HIP_MEMORY_SCOPE_AGENT);
          __hip_atomic_store(header_word(a.ws, HDR_DONE), 0, __ATOMIC_RELAXED,
                             __HIP_MEMORY_SCOPE_AGENT);
        }
      }
    }
  }
}

// Workspace of dlfp_append_attention_mixed_static: a fixed array in device
// memory, one copy per GPU the library runs on, held until the process ends.
// Host code must not pass the array's name to a kernel (on the host it only
// stands for the symbol); static_workspace() below looks up its device address
// once per device.
__device__ __align__(256) char scratch[DLFP_STATIC_WORKSPACE_BYTES];

__global__ void fill_zero_kernel(int* p, int64_t n) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i < n) p[i] = 0;
}

// Compute units of the current device (queried once per device).
int compute_units() {
  static int cached[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  if (!cached[dev]) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0)
      n = 256;
    cached[dev] = n;
  }
  return cached[dev];
}

constexpr int FUSED_APPEND_MAX_WGS = 16;

template <int G, bool APP, bool MIXED>
hipError_t launch(const Args& a, int grid, hipStream_t stream) {
  attention_mixed_kernel<G, APP, MIXED><<<grid, THREADS, 0, stream>>>(a);
  return hipGetLastError();
}

template <int G>
hipError_t launch_g(const Args& a, int grid, bool app, bool mixed, hipStream_t stream) {
  if (app)
    return mixed ? launch<G, true, true>(a, grid, stream) : launch<G, true, false>(a, grid, stream);
  return mixed ? launch<G, false, true>(a, grid, stream) : launch<G, false, false>(a, grid, stream);
}

// Validation, grid and launch shared by the entry points; `app` selects the
// fused append (k_new / v_new are ignored without it).  A batch without units
// returns DLFP_OK after its counts are checked, before any pointer is.
int launch_mixed(const dlfp_dims* dims, const dlfp_meta* meta, const int32_t* d_work,
                 const int32_t* d_block_table, int32_t max_blocks, int32_t num_blocks,
                 const void* q, bool app, const void* k_new, const void* v_new,
                 const void* k_cache,
                 const void* v_cache, float scale, void* out, int32_t out_dtype, void* workspace,
                 size_t workspace_bytes, hipStream_t stream) {
  int g = 0;
  const int st = dlfp::check_dims(dims, &g);
  if (st != DLFP_OK) return st;
  if (!meta) return DLFP_EINVAL;
  if (out_dtype != 0 && out_dtype != 1) return DLFP_EINVAL;
  if (!(scale > 0.f) || !(scale < 3.0e38f)) return DLFP_EINVAL;
  if (meta->num_units < 0 || meta->num_prefill_units < 0 ||
      meta->num_prefill_units > meta->num_units || meta->num_groups < 0)
    return DLFP_EINVAL;
  if (app && (meta->num_append < 0 || meta->num_waiting_units < 0 ||
              (meta->num_append > 0 && meta->num_waiting_units == 0) ||
              meta->num_waiting_units > meta->num_prefill_units))
    return DLFP_EINVAL;
  if (meta->num_units == 0) return DLFP_OK;
  if (meta->prefill_lead_units < 0 || meta->prefill_lead_units > meta->num_prefill_units ||
      (meta->decode_pages_in_flight != 1 && meta->decode_pages_in_flight != 2))
    return DLFP_EINVAL;
  if (!d_work || !d_block_table || !q || !k_cache || !v_cache || !out || !workspace)
    return DLFP_EINVAL;
  if (app && (!k_new || !v_new)) return DLFP_EINVAL;
  if (max_blocks <= 0 || num_blocks <= 0) return DLFP_EINVAL;
  if ((int64_t)workspace_bytes < meta->workspace_bytes ||
      workspace_bytes < (size_t)DLFP_WORKSPACE_PARTIALS)
    return DLFP_ENOSPC;
  if (meta->num_groups > DLFP_MAX_GROUPS) return DLFP_EINVAL;
  Args a;
  a.work = d_work;
  a.block_table = d_block_table;
  a.q = static_cast<const uint16_t*>(q);
  a.kc = static_cast<const uint16_t*>(k_cache);
  a.vc = static_cast<const uint16_t*>(v_cache);
  a.out = out;
  a.ws = static_cast<float*>(workspace);
  a.max_blocks = max_blocks;
  a.num_blocks = num_blocks;
  a.hq = dims->num_q_heads;
  a.hkv = dims->num_kv_heads;
  a.num_units = meta->num_units;
  a.num_prefill = meta->num_prefill_units;
  a.out_f32 = out_dtype;
  a.scale_log2 = scale * LOG2E;
  a.k_new = static_cast<const uint16_t*>(k_new);
  a.v_new = static_cast<const uint16_t*>(v_new);
  a.num_append = app ? meta->num_append : 0;
  a.num_waiting = app ? meta->num_waiting_units : 0;
  // Append workgroups in the launch: about two records per wavefront, a
  // multiple of 8.  Past FUSED_APPEND_MAX_WGS of them the records get a launch
  // of their own first: at the start of the attention launch each append
  // workgroup holds a CU slot, which pushes long prefill units to share CUs
  // (measured on Qwen3-0.6B shapes: chunks of 512-2048 prompt tokens took
  // 15-20% longer in one launch, while chunks of 64-256 gained 6-8% per
  // iteration from dropping the second launch).
  a.app_wgs = a.num_append > 0 ? (int)(((int64_t)a.num_append + 63) / 64 * 8) : 0;
  if (a.app_wgs > FUSED_APPEND_MAX_WGS) {
    Args r = a;
    r.app_wgs = (a.num_append + 3) / 4;
    r.num_waiting = 0;
    (void)hipGetLastError();
    append_records_kernel<<<r.app_wgs, THREADS, 0, stream>>>(r);
    if (hipGetLastError() != hipSuccess) return DLFP_EHIP;
    a.app_wgs = 0;
    a.num_append = 0;
    a.num_waiting = 0;
  }
  // Decode workgroups: enough to fill the resident slots of the device (two
  // per CU), fewer when there are fewer units; they drain the decode queue.
  // Only those that find a slot left by the append and prefill workgroups
  // from the start (at least 64) get units by position.
  const int cus = compute_units();
  const int decode_units = meta->num_units - meta->num_prefill_units;
  const int decode_wgs = std::min((decode_units + 3) / 4, 2 * cus);
  const int ahead = meta->num_prefill_units + a.app_wgs;
  const int slots = ahead < 2 * cus ? std::max(2 * cus - ahead, 64) : 2 * cus;
  a.decode_waves = 4 * decode_wgs;
  a.decode_static = std::min(decode_units, 4 * std::min(decode_wgs, slots));
  a.lead = meta->num_prefill_units;
  a.decode_lead = 0;
  a.deep = meta->decode_pages_in_flight == 2;
  if (meta->prefill_lead_units < meta->num_prefill_units && decode_wgs >= 8) {
    // the leading decode workgroups are resident from the start and take their
    // units by position; the ones after the other prefill units take tickets
    a.lead = meta->prefill_lead_units;
    a.decode_lead = std::min(decode_wgs, cus) / 8 * 8;
    a.decode_static = std::min(decode_units, 4 * a.decode_lead);
  }
  const int grid = a.app_wgs + meta->num_prefill_units + decode_wgs;
  const bool mixed = meta->num_prefill_units > 0 && decode_units > 0;
  (void)hipGetLastError();
  hipError_t e;
  switch (g) {
    case 1: e = launch_g<1>(a, grid, app, mixed, stream); break;
    case 2: e = launch_g<2>(a, grid, app, mixed, stream); break;
    case 4: e = launch_g<4>(a, grid, app, mixed, stream); break;
    default: e = launch_g<8>(a, grid, app, mixed, stream); break;
  }
  return e == hipSuccess ? DLFP_OK : DLFP_EHIP;
}

// Device address of `scratch` on the current device, looked up (and its
// header and counter region zeroed by a fill kernel on `stream`) on the first
// call for that device.  Launches leave the header and counters zero again.
int static_workspace(void** ptr, hipStream_t stream) {
  static std::mutex mu;
  static void* addr[64] = {nullptr};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return DLFP_EHIP;
  std::lock_guard<std::mutex> lock(mu);
  if (!addr[dev]) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) return DLFP_EHIP;
    const int64_t n = DLFP_WORKSPACE_PARTIALS / 4;
    (void)hipGetLastError();
    fill_zero_kernel<<<(unsigned)((n + 255) / 256), 256, 0, stream>>>(static_cast<int*>(p), n);
    if (hipGetLastError() != hipSuccess) return DLFP_EHIP;
    addr[dev] = p;
  }
  *ptr = addr[dev];
  return DLFP_OK;
}

}  // namespace

extern "C" int dlfp_attention_mixed(const dlfp_dims* dims, const dlfp_meta* meta,
                                    const int32_t* d_work,
                                    const int32_t* d_block_table, int32_t max_blocks,
                                    int32_t num_blocks, const void* q, const void* k_cache,
                                    const void* v_cache, float scale, void* out,
                                    int32_t out_dtype, void* workspace, size_t workspace_bytes,
                                    hipStream_t stream) {
  return launch_mixed(dims, meta, d_work, d_block_table, max_blocks, num_blocks, q, false,
                      nullptr, nullptr, k_cache, v_cache, scale, out, out_dtype, workspace,
                      workspace_bytes, stream);
}

extern "C" int dlfp_append_attention_mixed(const dlfp_dims* dims, const dlfp_meta* meta,
                                           const int32_t* d_work, const int32_t* d_block_table,
                                           int32_t max_blocks, int32_t num_blocks, const void* q,
                                           const void* k_new, const void* v_new, void* k_cache,
                                           void* v_cache, float scale, void* out,
                                           int32_t out_dtype, void* workspace,
                                           size_t workspace_bytes, hipStream_t stream) {
  return launch_mixed(dims, meta, d_work, d_block_table, max_blocks, num_blocks, q, true,
                      k_new, v_new, k_cache, v_cache, scale, out, out_dtype, workspace,
                      workspace_bytes, stream);
}

extern "C" int dlfp_append_attention_mixed_static(const dlfp_dims* dims, const dlfp_meta* meta,
                                                  const int32_t* d_work,
                                                  const int32_t* d_block_table,
                                                  int32_t max_blocks, int32_t num_blocks,
                                                  const void* q, const void* k_new,
                                                  const void* v_new, void* k_cache,
                                                  void* v_cache, float scale, void* out,
                                                  int32_t out_dtype, hipStream_t stream) {
  if (!meta) return DLFP_EINVAL;
  if (meta->workspace_bytes > (int64_t)DLFP_STATIC_WORKSPACE_BYTES) return DLFP_ENOSPC;
  if (meta->num_units == 0)  // checks the counts only; no set-up, no launch
    return launch_mixed(dims, meta, d_work, d_block_table, max_blocks, num_blocks, q, true,
                        k_new, v_new, k_cache, v_cache, scale, out, out_dtype, nullptr, 0,
                        stream);
  void* ws = nullptr;
  const int st = static_workspace(&ws, stream);
  if (st != DLFP_OK) return st;
  return launch_mixed(dims, meta, d_work, d_block_table, max_blocks, num_blocks, q, true, k_new,
                      v_new, k_cache, v_cache, scale, out, out_dtype, ws,
                      DLFP_STATIC_WORKSPACE_BYTES, stream);
}

extern "C" int dlfp_workspace_init(void* workspace, size_t workspace_bytes, hipStream_t stream) {
  if (!workspace) return DLFP_EINVAL;
  const int64_t bytes = DLFP_WORKSPACE_PARTIALS;
  if ((int64_t)workspace_bytes < bytes) return DLFP_ENOSPC;
  const int64_t n = bytes / 4;
  (void)hipGetLastError();
  fill_zero_kernel<<<(unsigned)((n + 255) / 256), 256, 0, stream>>>(static_cast<int*>(workspace),
                                                                     n);
  return hipGetLastError() == hipSuccess ? DLFP_OK : DLFP_EHIP;
}

extern "C" int dlfp_workspace_error(const void* workspace, int32_t* host_error,
                                    hipStream_t stream) {
  if (!workspace || !host_error) return DLFP_EINVAL;
  if (hipStreamSynchronize(stream) != hipSuccess) return DLFP_EHIP;
  if (hipMemcpy(host_error, workspace, sizeof(int32_t), hipMemcpyDeviceToHost) != hipSuccess)
    return DLFP_EHIP;
  return DLFP_OK;
}
