/*
 * dlfp.h -- C ABI of the mixed-iteration hot path of Decode-Latency Feedback
 * Prefill (DLFP) on AMD Instinct MI355X (gfx950).
 *
 * One mixed continuous-batching iteration (Eq. 1, Sec. 2.1) serves the set
 * D_t of decoding requests -- one new query token each -- together with p_t
 * prompt tokens admitted for chunked prefill, which attend causally to their
 * prompt's already-cached prefix plus the chunk itself (Sec. 2.1).  Keys and
 * values live in a paged cache addressed through per-sequence block tables
 * (PagedAttention, Sec. 2.1).  The iteration is:
 *
 *   dlfp_build_varlen_meta   host: packed-batch metadata and the work list
 *   dlfp_kv_append           device: write this iteration's K/V into pages
 *   dlfp_attention_mixed     device: ONE launch of attention for all rows
 *   dlfp_controller_step     host: Eq. 2 on the completion-timed latency
 *
 * dlfp_append_attention_mixed does the two device steps in one launch.
 *
 * The iteration latency that feeds the controller is the completion time of
 * the device work measured with HIP events (dlfp_timer_*), not the interval
 * between scheduler calls -- the proxy the paper identifies as the reason its
 * prototype failed to generalise (Sec. 3.2, Sec. 6.4, Sec. 11).
 *
 * Conventions for every call:
 *  - Return value: DLFP_OK (0) or a negative dlfp_status.  No call throws,
 *    aborts or prints.  No call synchronises a stream except two, by design:
 *    dlfp_timer_elapsed_ms waits for its stop event (completion timing) and
 *    dlfp_workspace_error synchronises the stream before reading the error
 *    word.  Every argument is validated before anything is launched; on a
 *    validation error nothing is launched and no output is written.  A
 *    DLFP_EHIP from a launch that follows another launch of the same call
 *    (only dlfp_append_attention_mixed with more than 128 append records,
 *    see there) leaves the first launch's work enqueued.
 *  - Empty batches: a launch call given no work (num_tokens 0 for
 *    dlfp_kv_append, a metadata with num_units 0 for the attention calls,
 *    as dlfp_build_varlen_meta makes for num_seqs 0) checks its dims and
 *    counts, launches nothing and returns DLFP_OK; its device pointers are
 *    not read and may be null (an empty device tensor's address).
 *  - Ownership: the caller owns every buffer (device and host).  The library
 *    allocates no device memory and keeps no pointer after returning.
 *  - Device calls are stream-ordered and asynchronous; a device-side fault
 *    surfaces at the caller's next synchronisation.  A failed launch is
 *    reported as DLFP_EHIP.
 *  - Supported shapes: head_dim 128, page 16 tokens, Hq = g * Hkv with
 *    g in {1, 2, 4, 8}; anything else is DLFP_EUNSUPPORTED.
 *
 * Device memory layouts (bf16 = IEEE bfloat16 stored as 16-bit words):
 *  - q           [num_tokens][Hq][128]        packed in cu_q order
 *  - k_new,v_new [num_tokens][Hkv][128]       this iteration's keys/values
 *  - k_cache     [num_blocks][Hkv][16][128]   key page: 16 token rows
 *  - v_cache     [num_blocks][Hkv][128][16]   value page: stored transposed,
 *                                             one 32-byte row per dimension;
 *                                             slot t sits at position
 *                                             pi(t), pi swapping slots 4-7
 *                                             with 8-11 (bits 2 and 3 of t)
 *  - block_table [num_seqs][max_blocks] int32 physical block of each page
 *  - out         [num_tokens][Hq][128]        bf16 or fp32
 *  Token j of sequence s lives in block block_table[s][j / 16], slot j % 16;
 *  its flat slot index is block * 16 + j % 16.
 */
#ifndef DLFP_H
#define DLFP_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define DLFP_HEAD_DIM 128
#define DLFP_PAGE_SIZE 16
/* Query rows (tokens x grouped query heads) held by one prefill unit. */
#define DLFP_TILE_ROWS 128
/* Longest key range of one work unit; the builder splits longer ranges.  A
 * unit keeps its slice of the block table in LDS, which bounds these. */
#define DLFP_MAX_DECODE_UNIT_KEYS 4096
#define DLFP_MAX_PREFILL_UNIT_KEYS 32768
/* int32 fields per work unit (see dlfp_build_varlen_meta). */
#define DLFP_WORK_INTS 16
/* Workspace layout: a 256-byte header (int32 word 0 = error flag, word
 * DLFP_WORKSPACE_TICKET_WORD = the decode queue's next ticket, word
 * DLFP_WORKSPACE_DONE_WORD = decode workgroups finished, word
 * DLFP_WORKSPACE_APPEND_WORD = append workgroups finished, word
 * DLFP_WORKSPACE_WAITED_WORD = prefill units past their wait for them; all
 * four are zero between launches), then a fixed region of DLFP_MAX_GROUPS int32 split
 * counters, then partial results from byte DLFP_WORKSPACE_PARTIALS on.  The
 * counter region has the same size for every launch, so one workspace can
 * serve iterations of any shape.  A launch that did not complete (a device
 * fault) leaves the header undefined: initialise the workspace again. */
#define DLFP_WORKSPACE_HEADER 256
#define DLFP_WORKSPACE_TICKET_WORD 16
#define DLFP_WORKSPACE_DONE_WORD 32
#define DLFP_WORKSPACE_APPEND_WORD 48
#define DLFP_WORKSPACE_WAITED_WORD 56
#define DLFP_MAX_GROUPS 65536
#define DLFP_WORKSPACE_PARTIALS (DLFP_WORKSPACE_HEADER + 4 * DLFP_MAX_GROUPS)

typedef enum {
  DLFP_OK = 0,
  DLFP_EINVAL = -1,        /* malformed argument (null pointer, negative size, bad value) */
  DLFP_ERANGE = -2,        /* index out of range (block id, sequence length vs table) */
  DLFP_ENOSPC = -3,        /* caller-provided capacity or workspace too small */
  DLFP_EHIP = -4,          /* a HIP runtime call or kernel launch failed */
  DLFP_EUNSUPPORTED = -5   /* shape outside the supported set */
} dlfp_status;

/* Attention shape of one layer. */
typedef struct {
  int32_t num_q_heads;   /* Hq */
  int32_t num_kv_heads;  /* Hkv; Hq / Hkv = g query heads share one KV head */
  int32_t head_dim;      /* must be 128 */
  int32_t page_size;     /* must be 16 */
} dlfp_dims;

/* How the attention launch splits key ranges (split-K).  Zero fields pick
 * the built-in policy.  Prefill: a launch too small to give every compute
 * unit a workgroup at 1024-key splits (decode workgroups counted) is
 * latency-bound and takes tiles of 32 rows (32 / g tokens) with the shortest
 * of 256, 512 or 1024-key splits that keeps its workgroups within two per
 * compute unit; otherwise, when the launch has a decode share, the prefill
 * takes the tallest tile of 128, 64 or 32 rows whose units, at the shortest
 * split of at least 1024 keys keeping them at most one per compute unit, come
 * within 1/16 of that count (32 rows when none does); a prefill share alone
 * takes 128-row tiles and the split (a multiple of 64 keys, at least 1024)
 * that minimises an estimate of the launch time.  The decode split is either
 * sqrt(256 W / F) keys for W decode keys over the F wavefronts of the
 * workgroup slots the prefill units leave (several queue rounds), or the
 * split that fits one round and best evens the decode workgroups over the
 * CUs, whichever an estimate of the launch time favours; a range longer than
 * its split is cut into equal parts, the last of them cut again into a half
 * and two quarters when the decode queue runs one to six rounds.  Grid
 * layout: when a launch has decode
 * units and more prefill units than compute units, one prefill unit per
 * compute unit leads the grid, then the decode workgroups (up to one per
 * compute unit), then the other prefill units, so that the memory-bound decode
 * share runs beside the matrix-core-bound prefill share from the start instead
 * of after it.  Decode page depth: two pages in flight in a launch without
 * prefill units, one beside them. */
typedef struct {
  int32_t decode_split_tokens;   /* keys per decode unit; 0 = auto, else a multiple of 16,
                                    at most DLFP_MAX_DECODE_UNIT_KEYS */
  int32_t prefill_split_tokens;  /* keys per prefill unit; 0 = auto, else a multiple of 64,
                                    at most DLFP_MAX_PREFILL_UNIT_KEYS */
  int32_t target_units;          /* wavefronts the device keeps resident for the attention
                                    launch, which the automatic split sizes are fitted to;
                                    0 = DLFP_DEFAULT_RESIDENT_WAVES */
  int32_t prefill_tile_tokens;   /* prompt tokens per prefill unit; 0 = auto, else at most
                                    DLFP_TILE_ROWS / g */
  int32_t prefill_lead_units;    /* grid layout of a launch with both shares: the number of
                                    prefill units placed before the first decode workgroups
                                    (the rest follow them); 0 = auto, -1 = all of them */
  int32_t decode_pages_in_flight;/* pages a decode wavefront keeps in flight beside its
                                    current one: 0 = auto, 1 or 2 */
} dlfp_tuning;

/* 256 compute units x 8 resident wavefronts (two 256-thread workgroups per CU). */
#define DLFP_DEFAULT_RESIDENT_WAVES 2048

/* Host-side metadata of one packed batch.  The caller provides the arrays and
 * their capacities; dlfp_build_varlen_meta fills arrays and counts. */
typedef struct {
  int32_t* cu_q;          /* [cap_seqs + 1] exclusive prefix sum of q_len */
  int32_t* q_pos0;        /* [cap_seqs] absolute position of each sequence's first new token */
  int32_t* slot_mapping;  /* [cap_tokens] flat pool slot of every new token, packed order */
  int32_t* work;          /* [cap_work][DLFP_WORK_INTS] work units, see below */
  int32_t cap_seqs, cap_tokens, cap_work;
  /* filled on success */
  int32_t num_seqs;
  int32_t num_tokens;         /* sum of q_len */
  int32_t num_units;          /* work units */
  int32_t num_prefill_units;  /* the first num_prefill_units units are prefill tiles */
  int32_t num_groups;         /* split groups (units sharing output rows) */
  int32_t decode_split_tokens, prefill_split_tokens;  /* splits actually used */
  int64_t workspace_bytes;    /* device workspace the attention launch needs */
  int32_t num_append;         /* append records stored after the units (see below) */
  int32_t num_waiting_units;  /* prefill units that read pages the append records write */
  int32_t prefill_lead_units; /* grid layout chosen (see dlfp_tuning); num_prefill_units
                                 when every prefill unit comes first */
  int32_t decode_pages_in_flight;  /* decode page depth chosen: 1 or 2 */
} dlfp_meta;

/* Work unit fields (int32 index into one DLFP_WORK_INTS record). */
enum {
  DLFP_W_SEQ = 0,      /* sequence */
  DLFP_W_KVHEAD = 1,   /* KV head; the unit serves its g query heads */
  DLFP_W_QTOK0 = 2,    /* first new token of the sequence the unit serves (0-based) */
  DLFP_W_QNTOK = 3,    /* number of new tokens it serves (1 for decode) */
  DLFP_W_KVBEGIN = 4,  /* first key (multiple of 16) */
  DLFP_W_KVEND = 5,    /* one past the last key */
  DLFP_W_GROUP = 6,    /* split group, -1 when the unit alone covers its rows */
  DLFP_W_SPLIT = 7,    /* index of this split within the group */
  DLFP_W_NSPLITS = 8,  /* splits in the group */
  DLFP_W_WSOFF = 9,    /* float offset of this unit's partial result in the workspace; a
                          slot holds O (rows x 128 floats), m[rows], l[rows] (rows = tokens x g),
                          padded to a multiple of 64 floats */
  DLFP_W_WSGROUP = 10, /* float offset of the group's split 0 partial */
  DLFP_W_KIND = 11,    /* DLFP_KIND_PREFILL, DLFP_KIND_DECODE or DLFP_KIND_APPEND */
  DLFP_W_QROW0 = 12,   /* packed row of the unit's first token in q and out:
                          cu_q[seq] + QTOK0 */
  DLFP_W_QPOS0 = 13,  /* position of the unit's first token: q_pos0[seq] + QTOK0 */
  DLFP_W_PAGE0 = 14,  /* decode units: block id of the unit's first page (KVBEGIN / 16) */
  DLFP_W_PAGE1 = 15   /* decode units: block id of its second page, -1 if it has one page */
};
enum { DLFP_KIND_PREFILL = 0, DLFP_KIND_DECODE = 1, DLFP_KIND_APPEND = 2 };

/* Build the metadata of one mixed iteration (Eq. 1's D_t and p_t, Sec. 2.1).
 *
 * num_seqs sequences, each with q_len[s] >= 1 new tokens (1 for a decoder,
 * the chunk size for a prefill slice) and kv_len[s] >= q_len[s] total keys
 * including the new ones.  block_table is the HOST copy [num_seqs][max_blocks];
 * every page a sequence uses must hold a block id in [0, num_blocks).
 *
 * Output (host arrays in *meta):
 *   cu_q[s]   = sum_{r<s} q_len[r];   q_pos0[s] = kv_len[s] - q_len[s]
 *   slot_mapping[cu_q[s] + i] = block_table[s][p / 16] * 16 + p % 16, p = q_pos0[s] + i
 *   work: prefill units (sequences with q_len > 1) first, one per
 *   (sequence, KV head, tile of at most DLFP_TILE_ROWS / g tokens, key split); then
 *   decode units (q_len == 1), one per (sequence, KV head, key split).
 *   Splits of the same rows form a group whose partial results the attention
 *   launch combines in split order.  After the num_units units follow
 *   num_append append records (KIND = DLFP_KIND_APPEND), read only by
 *   dlfp_append_attention_mixed: one per (prompt sequence, KV head, run of its
 *   new tokens inside one page), with SEQ, KVHEAD, QTOK0, QNTOK (1..16),
 *   QROW0 and QPOS0 as for units.  num_waiting_units counts the prefill units
 *   whose last key lies in a page holding a new token of their sequence.
 * Errors: DLFP_EINVAL (null pointers, q_len < 1, kv_len < q_len, bad tuning),
 * DLFP_ERANGE (a used page's block id outside [0, num_blocks) or beyond
 * max_blocks, or more than DLFP_MAX_GROUPS split groups), DLFP_ENOSPC (a capacity in *meta too small; the required counts
 * are still written to num_seqs / num_tokens / num_units / num_append; cap_work
 * must hold num_units + num_append records), DLFP_EUNSUPPORTED. */
int dlfp_build_varlen_meta(const dlfp_dims* dims, const dlfp_tuning* tuning, int32_t num_seqs,
                           const int32_t* q_len, const int32_t* kv_len,
                           const int32_t* block_table, int32_t max_blocks, int32_t num_blocks,
                           dlfp_meta* meta);

/* Write num_tokens new keys and values into their pages (PagedAttention cache
 * write, Sec. 2.1 and Sec. 3.2).  k_new/v_new: device bf16 [num_tokens][Hkv][128];
 * slot_mapping: device int32 [num_tokens] flat slots; caches as laid out above.
 * Slots outside [0, num_blocks * 16) are skipped (never written).  Bit copy. */
int dlfp_kv_append(const dlfp_dims* dims, int32_t num_tokens, const void* k_new,
                   const void* v_new, const int32_t* slot_mapping, void* k_cache, void* v_cache,
                   int32_t num_blocks, hipStream_t stream);

/* One launch of masked softmax attention for every new token of the batch
 * (the decode share and the prefill share of Eq. 1, Sec. 2.1).  For query
 * row i of sequence s at position p = q_pos0[s] + i and query head h, with
 * KV head h / g:  out = softmax_j(scale * q.k_j) v_j over keys j <= p.
 *
 * meta: the host metadata from dlfp_build_varlen_meta (only its counts are
 * read).  d_work, d_block_table: device copies of meta->work (each record
 * carries its sequence, rows, positions and key range; a decode unit's record
 * also carries the block ids of its first two pages) and of the block table
 * the metadata was built from.  q, k_cache, v_cache: device bf16.  out: device,
 * out_dtype 0 = bf16, 1 = fp32.  workspace: device scratch of at least
 * meta->workspace_bytes whose header and counter region (the first
 * DLFP_WORKSPACE_PARTIALS bytes) were zeroed once by dlfp_workspace_init;
 * every launch leaves the counters zero again.
 * Launches sharing one workspace must be stream-ordered.
 * Errors: DLFP_EINVAL, DLFP_ENOSPC (workspace too small), DLFP_EUNSUPPORTED,
 * DLFP_EHIP.  A block id outside [0, num_blocks) met on the device is not
 * read; the launch raises the workspace error word instead (dlfp_workspace_error). */
int dlfp_attention_mixed(const dlfp_dims* dims, const dlfp_meta* meta, const int32_t* d_work,
                         const int32_t* d_block_table, int32_t max_blocks, int32_t num_blocks,
                         const void* q, const void* k_cache, const void* v_cache, float scale,
                         void* out, int32_t out_dtype, void* workspace, size_t workspace_bytes,
                         hipStream_t stream);

/* dlfp_kv_append followed by dlfp_attention_mixed, as ONE launch (Sec. 2.1:
 * the iteration's cache write and its attention).  Arguments as for those two
 * calls; the slots written are the ones dlfp_build_varlen_meta derives from
 * the block table (its slot_mapping), d_work must hold the num_append append
 * records after the units, and k_cache/v_cache are written.  The result (out,
 * and every cache slot of a new token) equals that of the two calls; slots
 * that hold no new token are left as they were.
 *
 * Inside the launch a decode unit takes its own new key and value from k_new /
 * v_new and writes them to their slot.  The prompt tokens (the num_append
 * records) are written by the first workgroups of the grid -- 8 per 64
 * records; each writes its XCD's L2 back when done -- and count themselves
 * done on a workspace word; a prefill unit waits for that count, with a bounded poll,
 * before it loads the first page holding a new token.  The wait cannot hang:
 * a poll that runs out raises the workspace error word (value 2) and the
 * launch finishes with undefined output.  The last of the waiting prefill
 * units to finish zeroes the words again.  When the records would need more
 * than 16 such workgroups (above 128 records), they are written by a launch
 * of their own just before, and the prefill units do not wait.
 * Errors: as dlfp_attention_mixed.  With more than 128 append records, a
 * DLFP_EHIP reported for the attention launch can follow a successful enqueue
 * of the append-records launch: the cache may then hold the iteration's new
 * keys and values although the call failed (every argument is checked before
 * either launch, so only a runtime launch failure leads there). */
int dlfp_append_attention_mixed(const dlfp_dims* dims, const dlfp_meta* meta,
                                const int32_t* d_work, const int32_t* d_block_table,
                                int32_t max_blocks, int32_t num_blocks, const void* q,
                                const void* k_new, const void* v_new, void* k_cache,
                                void* v_cache, float scale, void* out, int32_t out_dtype,
                                void* workspace, size_t workspace_bytes, hipStream_t stream);

/* For callers that cannot allocate device memory: code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc.
 *
 * dlfp_append_attention_mixed with the workspace taken from a fixed array of
 * DLFP_STATIC_WORKSPACE_BYTES in device memory that the library holds, one
 * copy per GPU, until the process ends; arguments otherwise as for that call
 * (the caller still passes every input and output).  The call allocates
 * nothing: no hipMalloc, no hipFree, no allocating library routine.  Its first
 * call with work on a device looks up the array's address on that device and
 * zeroes its header and counter region with a fill kernel on `stream`; every
 * launch leaves them zero again.  All calls on one GPU share that GPU's array:
 * calls that overlap on one GPU (on different streams, or from different
 * threads without ordering) race on it and must not be made.
 * Errors: DLFP_ENOSPC when meta->workspace_bytes exceeds
 * DLFP_STATIC_WORKSPACE_BYTES (nothing is launched; a coarser split through
 * dlfp_tuning needs less), otherwise as dlfp_append_attention_mixed. */
#define DLFP_STATIC_WORKSPACE_BYTES (128u << 20)
int dlfp_append_attention_mixed_static(const dlfp_dims* dims, const dlfp_meta* meta,
                                       const int32_t* d_work, const int32_t* d_block_table,
                                       int32_t max_blocks, int32_t num_blocks, const void* q,
                                       const void* k_new, const void* v_new, void* k_cache,
                                       void* v_cache, float scale, void* out, int32_t out_dtype,
                                       hipStream_t stream);

/* Zero the workspace header and the whole counter region (the first
 * DLFP_WORKSPACE_PARTIALS bytes) with a stream-ordered fill kernel.  Needed
 * once per workspace allocation.  DLFP_ENOSPC if workspace_bytes is smaller. */
int dlfp_workspace_init(void* workspace, size_t workspace_bytes, hipStream_t stream);

/* Copy the workspace error word to *host_error after synchronising the stream:
 * 0 = no error, 1 = a block id outside the pool was met, 2 = a prefill unit of
 * dlfp_append_attention_mixed stopped waiting for the append records. */
int dlfp_workspace_error(const void* workspace, int32_t* host_error, hipStream_t stream);

/* Dense projection for the full-iteration latency of Eq. 1 (the linear
 * layers whose cost grows with the prefill chunk p_t, Sec. 2.1):
 *   out[i][j] = sum_l x[i][l] * w[j][l],  i < m, j < n, l < k
 * x: device bf16, row i at x + i * ldx (ldx >= k, a multiple of 8, x 16-byte
 * aligned); w: device bf16 [n][k] (one row per output feature, as a linear
 * layer's weight is stored), 16-byte aligned; out: device, row i at
 * out + i * ldo (ldo >= n, a multiple of 4), out_dtype 0 = bf16 (8-byte
 * aligned), 1 = fp32 (16-byte aligned).  fp32 accumulation.  n must be a
 * multiple of 128 and k of 64 (DLFP_EUNSUPPORTED otherwise); m = 0 launches
 * nothing.  Errors: DLFP_EINVAL, DLFP_EUNSUPPORTED, DLFP_EHIP. */
int dlfp_linear_bf16(int32_t m, int32_t n, int32_t k, const void* x, int32_t ldx, const void* w,
                     void* out, int32_t ldo, int32_t out_dtype, hipStream_t stream);

/* Proportional prefill-cap controller, Eq. 2 (Sec. 3.1):
 *   cap <- clamp(quantum * floor(cap * target / observed / quantum), c_min, c_max)
 * applied after each guarded cycle (at least one decoder and a prefill shared
 * it).  When the next cycle has no decoder the cap resets to c_initial and
 * prefill is uncapped (Sec. 3.1, Sec. 3.2).  Caller-owned plain struct. */
typedef struct {
  double target_ms;
  int32_t c_initial, c_min, c_max, quantum;
  int32_t cap;  /* current cap c_t */
} dlfp_controller;

/* Requires 0 < c_min <= c_initial <= c_max, quantum > 0, target_ms finite > 0. */
int dlfp_controller_init(dlfp_controller* ctrl, double target_ms, int32_t c_initial,
                         int32_t c_min, int32_t c_max, int32_t quantum);

/* After a cycle has COMPLETED: if last_was_guarded, update the cap from
 * observed_ms (the cycle's device completion time); then, if
 * num_decoding_next == 0, reset.  *next_cap receives the cap for the next
 * cycle's prefill, or -1 (uncapped) when no decoder is active.
 * DLFP_EINVAL if observed_ms is not finite and positive while
 * last_was_guarded (state unchanged). */
int dlfp_controller_step(dlfp_controller* ctrl, int32_t num_decoding_next,
                         int32_t last_was_guarded, double observed_ms, int32_t* next_cap);

/* Completion timer: a pair of HIP events around an iteration's device work.
 * The handle owns two events (no device memory). */
typedef struct dlfp_timer_s* dlfp_timer;
int dlfp_timer_create(dlfp_timer* timer);
int dlfp_timer_destroy(dlfp_timer timer);
int dlfp_timer_start(dlfp_timer timer, hipStream_t stream);
int dlfp_timer_stop(dlfp_timer timer, hipStream_t stream);
/* Block until the stop event has completed; elapsed device time in ms. */
int dlfp_timer_elapsed_ms(dlfp_timer timer, double* ms);

/* Enqueue on `stream` a one-wave kernel that idles for `microseconds` of
 * device wall-clock time (1..DLFP_MAX_HOLD_US; DLFP_EINVAL otherwise).  Call
 * it before dlfp_timer_start when the host enqueues an iteration's launches
 * one by one: they then run back to back and the timer sees device time only,
 * which is how one layer's share of an iteration's latency is measured.  The
 * kernel reads the wall clock and touches no memory; it always terminates. */
#define DLFP_MAX_HOLD_US 10000
int dlfp_stream_hold(int32_t microseconds, hipStream_t stream);

const char* dlfp_status_string(int status);

/* Library version, e.g. 100 for 0.1.0. */
int dlfp_version(void);

#ifdef __cplusplus
}
#endif

#endif /* DLFP_H */
