// Drives the host half of libdlfp (metadata builder and Eq. 2 controller) on
// seeded random inputs and prints every input and output as one JSON line per
// case, for tests/test_native_sanitized.py to check against the oracle twins.
// Built with a host compiler and AddressSanitizer + UndefinedBehaviorSanitizer,
// so any out-of-bounds access or undefined operation aborts the run.
//
// usage: host_driver SEED CASES
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <vector>

#include "dlfp.h"

namespace {

uint64_t g_state;
uint64_t next_u64() {  // splitmix64
  uint64_t z = (g_state += 0x9E3779B97F4A7C15ull);
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}
int64_t uniform(int64_t lo, int64_t hi) {  // inclusive
  return lo + (int64_t)(next_u64() % (uint64_t)(hi - lo + 1));
}

void print_array(const char* name, const int32_t* a, int64_t n) {
  std::printf("\"%s\":[", name);
  for (int64_t i = 0; i < n; ++i) std::printf(i ? ",%d" : "%d", a[i]);
  std::printf("],");
}

void meta_case(int id) {
  const int gs[] = {1, 2, 4, 8}, hkvs[] = {1, 2, 8};
  const int g = gs[uniform(0, 3)], hkv = hkvs[uniform(0, 2)];
  dlfp_dims dims = {g * hkv, hkv, 128, 16};
  dlfp_tuning tn = {0, 0, 0, 0};
  if (uniform(0, 1)) {
    tn.decode_split_tokens = (int32_t)(16 * uniform(0, 64));
    tn.prefill_split_tokens = (int32_t)(64 * uniform(0, 40));
    tn.prefill_tile_tokens = (int32_t)uniform(0, 128 / g);
  }
  const int n = (int)uniform(1, 24);
  std::vector<int32_t> q_len(n), kv_len(n);
  int max_pages = 1, total_pages = 0;
  for (int s = 0; s < n; ++s) {
    if (uniform(0, 9) < 7) {
      q_len[s] = 1;
      kv_len[s] = (int32_t)uniform(1, 3000);
    } else {
      q_len[s] = (int32_t)uniform(2, 1200);
      kv_len[s] = q_len[s] + (int32_t)uniform(0, 3000);
    }
    const int pages = (kv_len[s] + 15) / 16;
    max_pages = pages > max_pages ? pages : max_pages;
    total_pages += pages;
  }
  const int max_blocks = max_pages + (int)uniform(0, 3);
  const int num_blocks = total_pages + (int)uniform(0, 50);
  std::vector<int32_t> perm(num_blocks);
  for (int i = 0; i < num_blocks; ++i) perm[i] = i;
  for (int i = num_blocks - 1; i > 0; --i) std::swap(perm[i], perm[uniform(0, i)]);
  std::vector<int32_t> bt((size_t)n * max_blocks, -1);
  for (int s = 0, off = 0; s < n; ++s)
    for (int p = 0; p < (kv_len[s] + 15) / 16; ++p) bt[(size_t)s * max_blocks + p] = perm[off++];

  // capacity probe: nothing provided, counts still reported
  dlfp_meta probe = {};
  const int st0 = dlfp_build_varlen_meta(&dims, &tn, n, q_len.data(), kv_len.data(), bt.data(),
                                         max_blocks, num_blocks, &probe);
  const int records = probe.num_units + probe.num_append;
  std::vector<int32_t> cu_q(n + 1), q_pos0(n), slots(probe.num_tokens > 0 ? probe.num_tokens : 1),
      work((size_t)(records > 0 ? records : 1) * DLFP_WORK_INTS);
  dlfp_meta m = {};
  m.cu_q = cu_q.data();
  m.q_pos0 = q_pos0.data();
  m.slot_mapping = slots.data();
  m.work = work.data();
  m.cap_seqs = n;
  m.cap_tokens = probe.num_tokens;
  m.cap_work = records;
  const int st = dlfp_build_varlen_meta(&dims, &tn, n, q_len.data(), kv_len.data(), bt.data(),
                                        max_blocks, num_blocks, &m);
  std::printf("{\"kind\":\"meta\",\"case\":%d,\"hq\":%d,\"hkv\":%d,\"probe_status\":%d,"
              "\"status\":%d,\"tuning\":[%d,%d,%d,%d],\"max_blocks\":%d,\"num_blocks\":%d,",
              id, dims.num_q_heads, hkv, st0, st, tn.decode_split_tokens,
              tn.prefill_split_tokens, tn.target_units, tn.prefill_tile_tokens, max_blocks,
              num_blocks);
  print_array("q_len", q_len.data(), n);
  print_array("kv_len", kv_len.data(), n);
  print_array("bt", bt.data(), (int64_t)n * max_blocks);
  if (st == DLFP_OK) {
    print_array("cu_q", cu_q.data(), n + 1);
    print_array("q_pos0", q_pos0.data(), n);
    print_array("slots", slots.data(), m.num_tokens);
    print_array("work", work.data(), (int64_t)records * DLFP_WORK_INTS);
  }
  std::printf("\"num_units\":%d,\"num_prefill\":%d,\"num_groups\":%d,\"num_append\":%d,"
              "\"num_waiting\":%d,\"workspace_bytes\":%lld}\n",
              m.num_units, m.num_prefill_units, m.num_groups, m.num_append,
              m.num_waiting_units, (long long)m.workspace_bytes);

  // malformed inputs: one bad field each, expected status in the line
  std::vector<int32_t> bad_q = q_len, bad_bt = bt;
  bad_q[n - 1] = 0;
  bad_bt[(size_t)(n - 1) * max_blocks] = num_blocks;  // first page of the last sequence
  dlfp_tuning bad_tn = {17, 0, 0, 0};
  const int e_q = dlfp_build_varlen_meta(&dims, &tn, n, bad_q.data(), kv_len.data(), bt.data(),
                                         max_blocks, num_blocks, &m);
  const int e_bt = dlfp_build_varlen_meta(&dims, &tn, n, q_len.data(), kv_len.data(),
                                          bad_bt.data(), max_blocks, num_blocks, &m);
  const int e_tn = dlfp_build_varlen_meta(&dims, &bad_tn, n, q_len.data(), kv_len.data(),
                                          bt.data(), max_blocks, num_blocks, &m);
  const int e_nul = dlfp_build_varlen_meta(&dims, &tn, n, nullptr, kv_len.data(), bt.data(),
                                           max_blocks, num_blocks, &m);
  dlfp_dims bad_dims = {dims.num_q_heads, hkv, 64, 16};
  const int e_dim = dlfp_build_varlen_meta(&bad_dims, &tn, n, q_len.data(), kv_len.data(),
                                           bt.data(), max_blocks, num_blocks, &m);
  std::printf("{\"kind\":\"errors\",\"case\":%d,\"q_len_zero\":%d,\"block_out_of_pool\":%d,"
              "\"bad_tuning\":%d,\"null_q_len\":%d,\"head_dim_64\":%d}\n",
              id, e_q, e_bt, e_tn, e_nul, e_dim);
}

void controller_case(int id) {
  const int32_t c_min = (int32_t)(32 * uniform(1, 40)), c_max = c_min + (int32_t)(128 * uniform(0, 60));
  const int32_t c_init = (int32_t)uniform(c_min, c_max);
  const double target = 0.01 + (double)uniform(0, 100000) * 1e-3;
  dlfp_controller c;
  const int st = dlfp_controller_init(&c, target, c_init, c_min, c_max, 128);
  std::printf("{\"kind\":\"controller\",\"case\":%d,\"status\":%d,\"target\":%.17g,"
              "\"c_initial\":%d,\"c_min\":%d,\"c_max\":%d,\"steps\":[",
              id, st, target, c_init, c_min, c_max);
  for (int i = 0; i < 200; ++i) {
    const int nd = (int)uniform(0, 3), guarded = (int)uniform(0, 1);
    const double obs = target * (0.05 + (double)uniform(0, 100000) * 1e-4);
    int32_t next = 0;
    const int s = dlfp_controller_step(&c, nd, guarded, obs, &next);
    std::printf(i ? ",[%d,%d,%.17g,%d,%d]" : "[%d,%d,%.17g,%d,%d]", nd, guarded, obs, s, next);
  }
  int32_t next = 0;
  const int bad = dlfp_controller_step(&c, 1, 1, -1.0, &next);
  std::printf("],\"negative_observation\":%d}\n", bad);
}

}  // namespace

int main(int argc, char** argv) {
  if (argc != 3) return 2;
  g_state = std::strtoull(argv[1], nullptr, 10);
  const int cases = std::atoi(argv[2]);
  for (int i = 0; i < cases; ++i) {
    meta_case(i);
    controller_case(i);
  }
  return 0;
}
