// Host half of libdlfp: packed-batch metadata and work list, the Eq. 2
// controller, status strings.  Plain C++ (no HIP calls), so it also builds
// with a host compiler and its sanitizers.  Device launches live in the .hip
// sources; the completion timers in dlfp_timer.cpp.
#include <algorithm>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <limits>
#include <memory>
#include <vector>

#include "dlfp.h"
#include "dlfp_internal.h"

namespace {

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }
int64_t round_up(int64_t a, int64_t b) { return ceil_div(a, b) * b; }
// Prefill key ranges start on a 64-key tile.
constexpr int64_t KV_GRANULE_PREFILL = 64;

// Floats of one partial result: O (rows x 128), m[rows], l[rows], padded to 256 bytes.
int64_t slot_floats(int64_t rows) { return round_up(rows * (DLFP_HEAD_DIM + 2), 64); }

struct Unit {
  int32_t f[DLFP_WORK_INTS];
};
static_assert(sizeof(Unit) == DLFP_WORK_INTS * sizeof(int32_t), "work records are packed");

}  // namespace

namespace dlfp {

int check_dims(const dlfp_dims* dims, int* group) {
  if (!dims) return DLFP_EINVAL;
  if (dims->num_q_heads <= 0 || dims->num_kv_heads <= 0) return DLFP_EINVAL;
  if (dims->head_dim != DLFP_HEAD_DIM || dims->page_size != DLFP_PAGE_SIZE)
    return DLFP_EUNSUPPORTED;
  if (dims->num_q_heads % dims->num_kv_heads) return DLFP_EUNSUPPORTED;
  const int g = dims->num_q_heads / dims->num_kv_heads;
  if (g != 1 && g != 2 && g != 4 && g != 8) return DLFP_EUNSUPPORTED;
  if (group) *group = g;
  return DLFP_OK;
}

}  // namespace dlfp

extern "C" {

int dlfp_version(void) { return 100; }

const char* dlfp_status_string(int status) {
  switch (status) {
    case DLFP_OK: return "ok";
    case DLFP_EINVAL: return "invalid argument";
    case DLFP_ERANGE: return "index out of range";
    case DLFP_ENOSPC: return "capacity or workspace too small";
    case DLFP_EHIP: return "HIP runtime error";
    case DLFP_EUNSUPPORTED: return "unsupported shape";
    default: return "unknown status";
  }
}

// Work-list policy.  Prefill rows are packed token-major into tiles of
// DLFP_TILE_ROWS rows (DLFP_TILE_ROWS / g tokens, each with its g query heads
// that share one KV head).  Each tile's visible key range [0, last row's
// position] and each decoder's range [0, kv_len) is cut into equal splits when
// it is longer than the split size; splits of the same rows form a group that
// the attention launch combines in split order.  Prefill units are ordered
// KV-head-major (with workgroups dealt round-robin over the XCDs and the
// launch giving each XCD a contiguous range, units reading the same KV head
// share an L2), longest tile first within a head.
int dlfp_build_varlen_meta(const dlfp_dims* dims, const dlfp_tuning* tuning, int32_t num_seqs,
                           const int32_t* q_len, const int32_t* kv_len,
                           const int32_t* block_table, int32_t max_blocks, int32_t num_blocks,
                           dlfp_meta* meta) {
  int g = 0;
  int st = dlfp::check_dims(dims, &g);
  if (st != DLFP_OK) return st;
  if (!meta || num_seqs < 0) return DLFP_EINVAL;
  if (num_seqs > 0 && (!q_len || !kv_len || !block_table || max_blocks <= 0)) return DLFP_EINVAL;
  if (num_blocks < 0) return DLFP_EINVAL;
  dlfp_tuning tn = {0, 0, 0, 0, 0, 0};
  if (tuning) tn = *tuning;
  if (tn.prefill_lead_units < -1) return DLFP_EINVAL;
  if (tn.decode_pages_in_flight < 0 || tn.decode_pages_in_flight > 2) return DLFP_EINVAL;
  if (tn.decode_split_tokens < 0 || tn.decode_split_tokens % DLFP_PAGE_SIZE ||
      tn.decode_split_tokens > DLFP_MAX_DECODE_UNIT_KEYS)
    return DLFP_EINVAL;
  if (tn.prefill_split_tokens < 0 || tn.prefill_split_tokens % 64 ||
      tn.prefill_split_tokens > DLFP_MAX_PREFILL_UNIT_KEYS)
    return DLFP_EINVAL;
  if (tn.target_units < 0) return DLFP_EINVAL;
  if (tn.prefill_tile_tokens < 0 || tn.prefill_tile_tokens > DLFP_TILE_ROWS / g)
    return DLFP_EINVAL;
  const int64_t resident = tn.target_units ? tn.target_units : DLFP_DEFAULT_RESIDENT_WAVES;
  const int hkv = dims->num_kv_heads;
  int tile_tokens = tn.prefill_tile_tokens ? tn.prefill_tile_tokens : DLFP_TILE_ROWS / g;

  // Validate sequences and the pages they use.
  int64_t tokens = 0, pre_keys = 0;
  for (int s = 0; s < num_seqs; ++s) {
    const int32_t ql = q_len[s], kl = kv_len[s];
    if (ql < 1 || kl < ql) return DLFP_EINVAL;
    const int64_t pages = ceil_div(kl, DLFP_PAGE_SIZE);
    if (pages > max_blocks) return DLFP_ERANGE;
    const int32_t* row = block_table + (int64_t)s * max_blocks;
    int32_t lo = std::numeric_limits<int32_t>::max(), hi = std::numeric_limits<int32_t>::min();
    for (int64_t p = 0; p < pages; ++p) {  // branch-free, so the scan vectorises
      lo = std::min(lo, row[p]);
      hi = std::max(hi, row[p]);
    }
    if (lo < 0 || hi >= num_blocks) return DLFP_ERANGE;
    if ((int64_t)num_blocks * DLFP_PAGE_SIZE > std::numeric_limits<int32_t>::max())
      return DLFP_ERANGE;
    tokens += ql;
    if (ql > 1) {
      const int64_t pos0 = kl - ql;
      for (int64_t t0 = 0; t0 < ql; t0 += tile_tokens) {
        const int64_t nt = std::min<int64_t>(tile_tokens, ql - t0);
        pre_keys += (pos0 + t0 + nt) * hkv;
      }
    }
  }
  if (tokens > std::numeric_limits<int32_t>::max()) return DLFP_ERANGE;

  // Decode split for `slots` workgroup slots left by the prefill units
  // (F = 4 slots wavefronts; CUs = resident / 8).  Either the queue runs
  // several rounds: every unit then adds a fixed cost (query and block-table
  // loads, pipeline fill, its part of the merge) worth about 256 keys, the
  // split minimising work / F plus the longest unit is sqrt(256 W / F) keys
  // for W decode keys, and the launch lasts about units / F unit times plus
  // one (units of the last round start late and finish alone, slower than
  // when they shared the device).  Or the units fit in one round (at most F):
  // the launch then
  // lasts as long as the busiest CU, ceil(workgroups / min(CUs, slots)) units
  // of the longest length, so a split leaving some CUs two decode workgroups
  // and others one wastes half of the latter.  The one-round splits
  // (multiples of 16 keys from 128 up, in steps of about 6%) are weighed
  // against the sqrt split by these estimates; ties go to the longer split.
  int32_t max_kv = 0;
  int64_t dec_keys = 0;
  for (int s = 0; s < num_seqs; ++s)
    if (q_len[s] == 1) {
      max_kv = std::max(max_kv, kv_len[s]);
      dec_keys += (int64_t)kv_len[s] * hkv;
    }
  auto decode_split = [&](int64_t slots) -> int64_t {
    slots = std::max<int64_t>(1, slots);
    const int64_t free_waves = 4 * slots;
    const int64_t cu_cap = std::max<int64_t>(1, std::min<int64_t>(resident / 8, slots));
    auto units_and_longest = [&](int64_t sp, int64_t* longest) {
      int64_t n_units = 0;
      *longest = 0;
      for (int s = 0; s < num_seqs; ++s) {
        if (q_len[s] != 1) continue;
        const int64_t n = ceil_div(kv_len[s], sp);
        n_units += hkv * n;
        *longest = std::max(*longest, round_up(ceil_div(kv_len[s], n), DLFP_PAGE_SIZE));
      }
      return n_units;
    };
    const double root = std::sqrt(256.0 * (double)dec_keys / (double)free_waves);
    const int64_t s0 = std::clamp<int64_t>(round_up((int64_t)std::ceil(root), DLFP_PAGE_SIZE), 128,
                                           DLFP_MAX_DECODE_UNIT_KEYS);
    int64_t longest = 0;
    int64_t best_sp = s0;
    double best = std::numeric_limits<double>::infinity();
    const int64_t n0 = units_and_longest(s0, &longest);
    if (n0 > free_waves)
      best = ((double)n0 / (double)free_waves + 1.0) * (double)(longest + 256);
    const int64_t top = std::min<int64_t>(round_up(std::max<int32_t>(max_kv, 128), DLFP_PAGE_SIZE),
                                          DLFP_MAX_DECODE_UNIT_KEYS);
    for (int64_t sp = 128; sp <= top; sp = round_up(sp + std::max<int64_t>(16, sp / 16), 16)) {
      const int64_t n_units = units_and_longest(sp, &longest);
      if (n_units > free_waves) continue;
      const double e = (double)ceil_div(ceil_div(n_units, 4), cu_cap) * (double)(longest + 256);
      if (e <= best) {
        best = e;
        best_sp = sp;
      }
    }
    return best_sp;
  };
  // Prefill units of the iteration for a tile size and key split.
  auto prefill_units = [&](int64_t tt, int64_t split) {
    int64_t n = 0;
    for (int s = 0; s < num_seqs; ++s) {
      if (q_len[s] == 1) continue;
      const int64_t pos0 = kv_len[s] - q_len[s];
      for (int64_t t0 = 0; t0 < q_len[s]; t0 += tt)
        n += hkv * ceil_div(pos0 + t0 + std::min<int64_t>(tt, q_len[s] - t0), split);
    }
    return n;
  };
  // Prefill split.  Prefill alone: the split (multiples of 64 keys, at least
  // 1024) that minimises an estimate of the launch time, rounds x the time of
  // the busiest CU, in keys: a unit costs its longest part plus about 300 keys
  // of prologue, store and merge, and a CU running two units at once runs them
  // 1.11x faster than one after the other.  The longest part matters: a split
  // that leaves some tiles whole and cuts others in two makes the launch as
  // long as the whole ones.  (Fitted to Qwen3-0.6B/8B/32B last chunks, where
  // it picks the measured best: 0.6B 2048 tokens 143 against 175 us before,
  // 1024 tokens 83 against 102 us.)  A launch too small to give every CU a
  // workgroup at 1024-key splits (decode units counted four to a workgroup, at
  // the split they would take without prefill) is bound by the latency of its
  // longest unit and of the merge of its splits: its prefill takes tiles of
  // 32 rows (a merge then moves a quarter of the bytes) and the shortest split
  // of 256, 512 or 1024 keys that keeps all workgroups within the two a CU
  // holds.
  int64_t split_p = tn.prefill_split_tokens;
  int64_t dec_wgs0 = 0;
  {
    const int64_t sd0 = tn.decode_split_tokens ? tn.decode_split_tokens : decode_split(resident / 4);
    for (int s = 0; s < num_seqs; ++s)
      if (q_len[s] == 1) dec_wgs0 += hkv * ceil_div(kv_len[s], sd0);
    dec_wgs0 = ceil_div(dec_wgs0, 4);
  }
  if (!split_p && !tn.prefill_tile_tokens && pre_keys > 0 &&
      prefill_units(tile_tokens, 1024) + dec_wgs0 < resident / 8) {
    const int small = std::max(1, 32 / g);
    for (int64_t sp : {256, 512, 1024}) {
      if (prefill_units(small, sp) + dec_wgs0 <= resident / 4) {
        tile_tokens = small;
        split_p = sp;
        break;
      }
    }
  }
  // Beside a decode share the prefill units wait on loaded memory and their
  // split merges are on the launch's critical path: the units should number
  // about one per compute unit (more leave decode workgroups without a slot,
  // fewer leave long key loops), each as tall as that allows (a shorter tile
  // re-reads its keys and values more often but merges fewer bytes per row
  // group).  So the tallest tile of 128, 64 or 32 rows whose units, with the
  // shortest split of at least 1024 keys that keeps them at most one per
  // compute unit, come within 1/16 of that count; else 32 rows.  (Measured on
  // Qwen3-0.6B shapes beside 32 decoders: 44-48 us per layer instead of
  // 50-54 us for chunks of 64-256 tokens over prefixes of 2-6k keys.)
  const bool has_decode = dec_keys > 0;
  if (!split_p && !tn.prefill_tile_tokens && pre_keys > 0 && has_decode) {
    const int64_t target = std::max<int64_t>(1, resident / 8);
    for (int rows : {DLFP_TILE_ROWS, DLFP_TILE_ROWS / 2, DLFP_TILE_ROWS / 4}) {
      const int64_t tt = std::max(1, rows / g);
      // The shortest split of 1024 + 64 k keys keeping the units within the
      // target (DLFP_MAX_PREFILL_UNIT_KEYS when none does), by bisection: the
      // unit count only falls as the split grows.
      int64_t lo = 0, hi = (DLFP_MAX_PREFILL_UNIT_KEYS - 1024) / 64;
      while (lo < hi) {
        const int64_t mid = (lo + hi) / 2;
        if (prefill_units(tt, 1024 + 64 * mid) > target)
          lo = mid + 1;
        else
          hi = mid;
      }
      const int64_t sp = 1024 + 64 * lo;
      if (prefill_units(tt, sp) * 16 >= target * 15 || rows == DLFP_TILE_ROWS / 4) {
        tile_tokens = (int)tt;
        split_p = sp;
        break;
      }
    }
  }
  if (!split_p) {
    const int64_t cus = std::max<int64_t>(1, resident / 8), slots = 2 * cus;
    int64_t max_kend = 0;
    for (int s = 0; s < num_seqs; ++s)
      if (q_len[s] != 1) max_kend = std::max<int64_t>(max_kend, kv_len[s]);
    double best = std::numeric_limits<double>::infinity();
    for (int64_t sp = 1024;; sp += 64) {
      int64_t n = 0, longest = 0;
      for (int s = 0; s < num_seqs; ++s) {
        if (q_len[s] == 1) continue;
        const int64_t pos0 = kv_len[s] - q_len[s];
        for (int64_t t0 = 0; t0 < q_len[s]; t0 += tile_tokens) {
          const int64_t kend = pos0 + t0 + std::min<int64_t>(tile_tokens, q_len[s] - t0);
          const int64_t part = round_up(ceil_div(kend, ceil_div(kend, sp)), KV_GRANULE_PREFILL);
          n += hkv * ceil_div(kend, part);
          longest = std::max(longest, part);
        }
      }
      const double unit = 300.0 + (double)longest;
      const double e = (double)ceil_div(n, slots) * (n > cus ? 2.0 * (300.0 + longest / 1.11) : unit);
      if (e < best) {
        best = e;
        split_p = sp;
      }
      if (sp >= max_kend || sp >= DLFP_MAX_PREFILL_UNIT_KEYS) break;
    }
  }
  int64_t split_d = tn.decode_split_tokens;
  if (!split_d) {
    int64_t pre_units = 0;
    for (int s = 0; s < num_seqs; ++s) {
      if (q_len[s] == 1) continue;
      const int64_t pos0 = kv_len[s] - q_len[s];
      for (int64_t t0 = 0; t0 < q_len[s]; t0 += tile_tokens) {
        const int64_t nt = std::min<int64_t>(tile_tokens, q_len[s] - t0);
        pre_units += hkv * ceil_div(pos0 + t0 + nt, split_p);
      }
    }
    // The decode share starts in the workgroup slots (two per CU, four
    // wavefronts each) that the prefill units leave, at least 64; when the
    // prefill units take them all, it runs as they retire.
    split_d = decode_split(pre_units < resident / 4
                               ? std::max<int64_t>(resident / 4 - pre_units, 64)
                               : resident / 4);
  }

  // Build units: prefill (KV-head-major), then decode.  Capacity: every key
  // range is cut into at most ceil(range / split) parts, plus two tail pieces.
  std::vector<Unit> units;
  {
    int64_t bound = 0;
    for (int s = 0; s < num_seqs; ++s) {
      if (q_len[s] == 1) {
        bound += hkv * (ceil_div(kv_len[s], split_d) + 2);
        continue;
      }
      const int64_t pos0 = kv_len[s] - q_len[s];
      for (int64_t t0 = 0; t0 < q_len[s]; t0 += tile_tokens)
        bound += hkv * (ceil_div(pos0 + t0 + std::min<int64_t>(tile_tokens, q_len[s] - t0),
                                 split_p) + 2);
    }
    units.reserve((size_t)bound);
  }
  std::vector<int64_t> cu_q_of(num_seqs + 1, 0);  // packed row of each sequence's first token
  for (int s = 0; s < num_seqs; ++s) cu_q_of[s + 1] = cu_q_of[s] + q_len[s];
  int32_t groups = 0;
  std::vector<int64_t> group_rows;  // rows of each group
  // A key range longer than the split is cut into equal parts (rounded up
  // to the granule), so the units of a group finish together.
  // With `tail`, the last part is cut again into a half and two quarters
  // (decode units that run in several queue rounds: the queue hands out the
  // longest units first, so these short pieces even out the end of the launch).
  std::vector<int64_t> cut;
  auto emit = [&](int s, int kh, int64_t t0, int64_t nt, int64_t kend, int64_t split,
                  int64_t granule, int kind, bool tail = false) {
    int64_t nsp = ceil_div(kend, split);
    const int64_t part = round_up(ceil_div(kend, nsp), granule);
    nsp = ceil_div(kend, part);
    cut.clear();
    for (int64_t j = 0; j < nsp; ++j) cut.push_back(j * part);
    if (tail) {
      const int64_t b = (nsp - 1) * part, len = kend - b;
      const int64_t h = round_up(ceil_div(len, 2), granule), q = round_up(ceil_div(len - h, 2), granule);
      if (len >= 4 * granule && h < len && h + q < len) {
        cut.push_back(b + h);
        cut.push_back(b + h + q);
      }
    }
    cut.push_back(kend);
    nsp = (int64_t)cut.size() - 1;
    const int32_t grp = nsp > 1 ? groups++ : -1;
    if (nsp > 1) group_rows.push_back(nt * g);
    for (int64_t j = 0; j < nsp; ++j) {
      Unit u;
      std::memset(&u, 0, sizeof(u));
      u.f[DLFP_W_SEQ] = s;
      u.f[DLFP_W_KVHEAD] = kh;
      u.f[DLFP_W_QTOK0] = (int32_t)t0;
      u.f[DLFP_W_QNTOK] = (int32_t)nt;
      u.f[DLFP_W_KVBEGIN] = (int32_t)cut[j];
      u.f[DLFP_W_KVEND] = (int32_t)cut[j + 1];
      u.f[DLFP_W_GROUP] = grp;
      u.f[DLFP_W_SPLIT] = (int32_t)j;
      u.f[DLFP_W_NSPLITS] = (int32_t)nsp;
      u.f[DLFP_W_KIND] = kind;
      u.f[DLFP_W_QROW0] = (int32_t)(cu_q_of[s] + t0);
      u.f[DLFP_W_QPOS0] = (int32_t)(kv_len[s] - q_len[s] + t0);
      if (kind == DLFP_KIND_DECODE) {
        // The unit's first two block ids travel with the record, so its first
        // page loads go out with its query and block-table loads.
        const int32_t* row = block_table + (int64_t)s * max_blocks;
        const int64_t pg = u.f[DLFP_W_KVBEGIN] / DLFP_PAGE_SIZE;
        const int64_t last = (u.f[DLFP_W_KVEND] - 1) / DLFP_PAGE_SIZE;
        u.f[DLFP_W_PAGE0] = row[pg];
        u.f[DLFP_W_PAGE1] = pg + 1 <= last ? row[pg + 1] : -1;
      }
      units.push_back(u);
    }
  };
  // Prefill tiles of one KV head go longest first, so that the workgroups of
  // an XCD (which takes a contiguous range of prefill units) start the long
  // tiles early.
  struct Tile {
    int s;
    int64_t t0, nt, kend;
  };
  std::vector<Tile> tiles;
  for (int kh = 0; kh < hkv; ++kh) {
    tiles.clear();
    for (int s = 0; s < num_seqs; ++s) {
      if (q_len[s] == 1) continue;
      const int64_t pos0 = kv_len[s] - q_len[s];
      for (int64_t t0 = 0; t0 < q_len[s]; t0 += tile_tokens) {
        const int64_t nt = std::min<int64_t>(tile_tokens, q_len[s] - t0);
        tiles.push_back(Tile{s, t0, nt, pos0 + t0 + nt});
      }
    }
    std::stable_sort(tiles.begin(), tiles.end(),
                     [](const Tile& x, const Tile& y) { return x.kend > y.kend; });
    for (const Tile& t : tiles)
      emit(t.s, kh, t.t0, t.nt, t.kend, split_p, KV_GRANULE_PREFILL, DLFP_KIND_PREFILL);
  }
  const int64_t num_prefill = (int64_t)units.size();
  // Decode units that run in a few queue rounds (more units than the wavefronts
  // the prefill units leave, but not so many that the last round is a small
  // part of the launch anyway) get the short tail pieces.
  bool decode_tail = false;
  if (!tn.decode_split_tokens) {
    int64_t n_dec = 0;
    for (int s = 0; s < num_seqs; ++s)
      if (q_len[s] == 1) n_dec += hkv * ceil_div(kv_len[s], split_d);
    const int64_t slots_d = num_prefill < resident / 4
                                ? std::max<int64_t>(resident / 4 - num_prefill, 64) : resident / 4;
    decode_tail = n_dec > 4 * slots_d && n_dec <= 24 * slots_d;
  }
  for (int s = 0; s < num_seqs; ++s) {
    if (q_len[s] != 1) continue;
    for (int kh = 0; kh < hkv; ++kh)
      emit(s, kh, 0, 1, kv_len[s], split_d, DLFP_PAGE_SIZE, DLFP_KIND_DECODE, decode_tail);
  }
  // Decode wavefronts take units in list order from a queue: longest first,
  // ties in emission order (a stable counting sort on the key count, which the
  // split keeps within 1..DLFP_MAX_DECODE_UNIT_KEYS).
  {
    constexpr int32_t K = DLFP_MAX_DECODE_UNIT_KEYS;
    const size_t first = (size_t)num_prefill, nd = units.size() - first;
    std::vector<int32_t> start(K + 1, 0);
    for (size_t i = first; i < units.size(); ++i) {
      const int32_t len = units[i].f[DLFP_W_KVEND] - units[i].f[DLFP_W_KVBEGIN];
      if (len < 1 || len > K) return DLFP_ERANGE;
      ++start[K - len + 1];
    }
    for (int32_t b = 1; b <= K; ++b) start[b] += start[b - 1];
    std::unique_ptr<Unit[]> sorted(new Unit[nd]);  // no zero fill: every slot is written
    for (size_t i = first; i < units.size(); ++i) {
      const int32_t len = units[i].f[DLFP_W_KVEND] - units[i].f[DLFP_W_KVBEGIN];
      sorted[start[K - len]++] = units[i];
    }
    std::copy(sorted.get(), sorted.get() + nd, units.begin() + first);
  }
  if ((int64_t)units.size() > std::numeric_limits<int32_t>::max() / DLFP_WORK_INTS)
    return DLFP_ERANGE;
  if (groups > DLFP_MAX_GROUPS) return DLFP_ERANGE;

  // Workspace: header, the fixed counter region, then partial slots.
  const int64_t partial_base_bytes = DLFP_WORKSPACE_PARTIALS;
  std::vector<int64_t> group_off(groups, 0);
  int64_t off = partial_base_bytes / 4;
  {
    // assign in order of first appearance
    std::vector<int64_t> seen(groups, -1);
    for (const Unit& u : units) {
      const int32_t grp = u.f[DLFP_W_GROUP];
      if (grp < 0 || seen[grp] >= 0) continue;
      seen[grp] = off;
      group_off[grp] = off;
      off += (int64_t)u.f[DLFP_W_NSPLITS] * slot_floats(group_rows[grp]);
    }
  }
  if (off > std::numeric_limits<int32_t>::max()) return DLFP_ERANGE;
  for (Unit& u : units) {
    const int32_t grp = u.f[DLFP_W_GROUP];
    if (grp < 0) continue;
    const int64_t slot = slot_floats(group_rows[grp]);
    u.f[DLFP_W_WSGROUP] = (int32_t)group_off[grp];
    u.f[DLFP_W_WSOFF] = (int32_t)(group_off[grp] + u.f[DLFP_W_SPLIT] * slot);
  }

  // Append records for the one-launch cache write: each prompt sequence's new
  // tokens cut at page boundaries, per KV head (decode units write their own
  // token).  A prefill unit waits for them when its last key lies in a page
  // from the one holding its sequence's first new token on.
  std::vector<Unit> appends;
  {
    int64_t n = 0;
    for (int s = 0; s < num_seqs; ++s)
      if (q_len[s] != 1) n += hkv * (q_len[s] / DLFP_PAGE_SIZE + 2);
    appends.reserve((size_t)n);
  }
  for (int s = 0; s < num_seqs; ++s) {
    if (q_len[s] == 1) continue;
    const int64_t pos0 = kv_len[s] - q_len[s];
    for (int kh = 0; kh < hkv; ++kh)
      for (int64_t p = pos0; p < kv_len[s];) {
        const int64_t n = std::min<int64_t>(DLFP_PAGE_SIZE - p % DLFP_PAGE_SIZE, kv_len[s] - p);
        Unit u;
        std::memset(&u, 0, sizeof(u));
        u.f[DLFP_W_SEQ] = s;
        u.f[DLFP_W_KVHEAD] = kh;
        u.f[DLFP_W_QTOK0] = (int32_t)(p - pos0);
        u.f[DLFP_W_QNTOK] = (int32_t)n;
        u.f[DLFP_W_KVBEGIN] = (int32_t)p;
        u.f[DLFP_W_KVEND] = (int32_t)(p + n);
        u.f[DLFP_W_GROUP] = -1;
        u.f[DLFP_W_NSPLITS] = 1;
        u.f[DLFP_W_KIND] = DLFP_KIND_APPEND;
        u.f[DLFP_W_QROW0] = (int32_t)(cu_q_of[s] + p - pos0);
        u.f[DLFP_W_QPOS0] = (int32_t)p;
        appends.push_back(u);
        p += n;
      }
  }
  int64_t waiting = 0;
  for (int64_t i = 0; i < num_prefill; ++i) {
    const Unit& u = units[i];
    const int64_t pos0 = u.f[DLFP_W_QPOS0] - u.f[DLFP_W_QTOK0];
    if ((u.f[DLFP_W_KVEND] - 1) / DLFP_PAGE_SIZE >= pos0 / DLFP_PAGE_SIZE) ++waiting;
  }
  const int64_t records = (int64_t)(units.size() + appends.size());
  if (records > std::numeric_limits<int32_t>::max() / DLFP_WORK_INTS) return DLFP_ERANGE;

  meta->num_seqs = num_seqs;
  meta->num_tokens = (int32_t)tokens;
  meta->num_units = (int32_t)units.size();
  meta->num_prefill_units = (int32_t)num_prefill;
  meta->num_groups = groups;
  meta->decode_split_tokens = (int32_t)split_d;
  meta->prefill_split_tokens = (int32_t)split_p;
  meta->workspace_bytes = std::max<int64_t>(off * 4, partial_base_bytes);
  meta->num_append = (int32_t)appends.size();
  meta->num_waiting_units = (int32_t)waiting;
  // Grid layout: with more prefill units than compute units, one per compute
  // unit leads and the decode workgroups follow, so the two shares run side by
  // side from the start instead of the decode units running alone after the
  // last prefill tile.
  const int64_t n_dec_units = (int64_t)units.size() - num_prefill;
  const int64_t cus = std::max<int64_t>(1, resident / 8);
  int64_t lead = num_prefill;
  if (tn.prefill_lead_units > 0)
    lead = std::min<int64_t>(tn.prefill_lead_units, num_prefill);
  else if (tn.prefill_lead_units == 0 && n_dec_units > 0 && num_prefill > cus)
    lead = cus;
  meta->prefill_lead_units = (int32_t)lead;
  // Decode page depth: two pages in flight without a prefill share; beside
  // one, one page (deeper decode queues delay the prefill tiles' loads; on the
  // Qwen3-32B sweep a second page gained nothing at p_t <= 1024 and lost 3-5%
  // at larger chunks).
  const int depth = tn.decode_pages_in_flight ? tn.decode_pages_in_flight
                                              : (num_prefill == 0 ? 2 : 1);
  meta->decode_pages_in_flight = depth;
  if (meta->cap_seqs < num_seqs || meta->cap_tokens < tokens || meta->cap_work < records)
    return DLFP_ENOSPC;
  if ((num_seqs > 0 && (!meta->cu_q || !meta->q_pos0)) || (tokens > 0 && !meta->slot_mapping) ||
      (records > 0 && !meta->work))
    return DLFP_EINVAL;
  if (meta->cu_q) meta->cu_q[0] = 0;
  int64_t t = 0;
  for (int s = 0; s < num_seqs; ++s) {
    const int32_t pos0 = kv_len[s] - q_len[s];
    meta->q_pos0[s] = pos0;
    const int32_t* row = block_table + (int64_t)s * max_blocks;
    for (int32_t i = 0; i < q_len[s]; ++i) {
      const int32_t p = pos0 + i;
      meta->slot_mapping[t++] = row[p / DLFP_PAGE_SIZE] * DLFP_PAGE_SIZE + p % DLFP_PAGE_SIZE;
    }
    meta->cu_q[s + 1] = (int32_t)t;
  }
  if (!units.empty()) std::memcpy(meta->work, units.data(), units.size() * sizeof(Unit));
  if (!appends.empty())
    std::memcpy(meta->work + units.size() * DLFP_WORK_INTS, appends.data(),
                appends.size() * sizeof(Unit));
  return DLFP_OK;
}

int dlfp_controller_init(dlfp_controller* ctrl, double target_ms, int32_t c_initial,
                         int32_t c_min, int32_t c_max, int32_t quantum) {
  if (!ctrl) return DLFP_EINVAL;
  if (!(std::isfinite(target_ms) && target_ms > 0.0)) return DLFP_EINVAL;
  if (!(0 < c_min && c_min <= c_initial && c_initial <= c_max) || quantum <= 0)
    return DLFP_EINVAL;
  ctrl->target_ms = target_ms;
  ctrl->c_initial = c_initial;
  ctrl->c_min = c_min;
  ctrl->c_max = c_max;
  ctrl->quantum = quantum;
  ctrl->cap = c_initial;
  return DLFP_OK;
}

// Eq. 2 (Sec. 3.1).  floor_quantum(x) = quantum * floor(x / quantum) in
// double precision, then clamp to [c_min, c_max].
int dlfp_controller_step(dlfp_controller* ctrl, int32_t num_decoding_next,
                         int32_t last_was_guarded, double observed_ms, int32_t* next_cap) {
  if (!ctrl || !next_cap || num_decoding_next < 0) return DLFP_EINVAL;
  if (last_was_guarded) {
    if (!(std::isfinite(observed_ms) && observed_ms > 0.0)) return DLFP_EINVAL;
    const double x = (double)ctrl->cap * ctrl->target_ms / observed_ms;
    const double q = std::floor(x / ctrl->quantum);
    int64_t c;
    if (!(q < (double)std::numeric_limits<int32_t>::max()))
      c = ctrl->c_max;
    else
      c = (int64_t)q * ctrl->quantum;
    c = std::min<int64_t>(std::max<int64_t>(c, ctrl->c_min), ctrl->c_max);
    ctrl->cap = (int32_t)c;
  }
  if (num_decoding_next == 0) {
    ctrl->cap = ctrl->c_initial;
    *next_cap = -1;
  } else {
    *next_cap = ctrl->cap;
  }
  return DLFP_OK;
}

}  // extern "C"
