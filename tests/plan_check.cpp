// Host-planner driver for the address and undefined-behaviour sanitizers.
// Builds with g++ alone (no HIP): exercises laminar_plan_create and
// laminar_plan_create_cascade over random and edge-case batches, checks that
// every (trajectory, kv-head, page) is covered exactly once, and frees every
// plan.
#include <cstdio>
#include <cstdlib>
#include <random>
#include <vector>

#include "laminar_decode_attn.h"

static int fail(const char* what) {
  std::printf("plan_check FAIL: %s\n", what);
  return 1;
}

static int check(const std::vector<int32_t>& lens, int hkv, int ppi, int waves,
                 const std::vector<int32_t>* group_of = nullptr,
                 const std::vector<int32_t>* group_pages = nullptr) {
  laminar_attn_desc d = {};
  d.batch = int32_t(lens.size());
  d.num_q_heads = hkv * 4;
  d.num_kv_heads = hkv;
  d.head_dim = 128;
  d.page_size = 16;
  d.num_pages = 1 << 30;
  d.max_blocks_per_seq = 8192;
  d.kv_dtype = LAMINAR_KV_BF16;
  d.softmax_scale = 0.125f;
  d.pages_per_item = ppi;
  d.waves_per_item = waves;
  laminar_plan* p = nullptr;
  const laminar_status st =
      group_of ? laminar_plan_create_cascade(
                     &d, lens.data(), group_of->data(),
                     int32_t(group_pages->size()), group_pages->data(), 256, &p)
               : laminar_plan_create(&d, lens.data(), 256, &p);
  if (st != LAMINAR_OK || !p) return fail("create");
  const int nc = laminar_plan_num_cascade_units(p);
  const int nm = laminar_plan_num_cascade_members(p);
  std::vector<int32_t> cunits(size_t(4) * (nc > 0 ? nc : 1));
  std::vector<int32_t> cmem(size_t(2) * (nm > 0 ? nm : 1));
  if (laminar_plan_cascade_units_copy(p, cunits.data(), nc) != nc ||
      laminar_plan_cascade_members_copy(p, cmem.data(), nm) != nm)
    return fail("cascade copy");
  const int n = laminar_plan_num_items(p);
  std::vector<int32_t> items(size_t(4) * (n > 0 ? n : 1));
  if (laminar_plan_items_copy(p, items.data(), n) != n) return fail("copy");
  std::vector<std::vector<char>> seen(lens.size() * hkv);
  for (size_t u = 0; u < seen.size(); ++u)
    seen[u].assign((lens[u / hkv] + 15) / 16, 0);
  for (int i = 0; i < n; ++i) {
    const int unit = items[4 * i], p0 = items[4 * i + 1], p1 = items[4 * i + 2];
    if (unit < 0) {                       // cascade item: every member
      const int cu = -unit - 1;
      if (cu >= nc) return fail("cascade unit");
      const int cnt = cunits[4 * cu + 1], moff = cunits[4 * cu + 2];
      const int kvh = cunits[4 * cu + 3];
      if (moff < 0 || moff + cnt > nm || kvh < 0 || kvh >= hkv)
        return fail("cascade header");
      for (int j = 0; j < cnt; ++j) {
        const size_t u = size_t(cmem[2 * (moff + j)]) * hkv + kvh;
        if (u >= seen.size() || p0 < 0 || p0 > p1) return fail("cascade member");
        for (int q = p0; q < p1 && q < int(seen[u].size()); ++q) {
          if (seen[u][q]) return fail("double cover (cascade)");
          seen[u][q] = 1;
        }
      }
      continue;
    }
    if (size_t(unit) >= seen.size()) return fail("unit");
    if (p0 < 0 || p1 > int(seen[unit].size()) || p0 > p1) return fail("range");
    for (int q = p0; q < p1; ++q) {
      if (seen[unit][q]) return fail("double cover");
      seen[unit][q] = 1;
    }
  }
  for (auto& v : seen)
    for (char c : v)
      if (!c) return fail("hole");
  const int m = laminar_plan_num_merges(p);
  std::vector<int32_t> merges(size_t(4) * (m > 0 ? m : 1));
  if (laminar_plan_merges_copy(p, merges.data(), m) != m) return fail("merges");
  laminar_plan_destroy(p);
  return 0;
}

int main() {
  std::mt19937 rng(7);
  std::lognormal_distribution<double> len_dist(7.0, 1.5);
  for (int trial = 0; trial < 200; ++trial) {
    const int b = 1 + int(rng() % 400);
    std::vector<int32_t> lens(b);
    for (auto& l : lens) {
      double x = len_dist(rng);
      l = x > 98304 ? 98304 : int32_t(x);
      if (rng() % 20 == 0) l = 0;
    }
    const int hkv = 1 << (rng() % 4);
    const int ppis[] = {0, 1, 2, 7, 64, 1 << 20};
    const int waves[] = {0, 1, 2, 4};
    if (check(lens, hkv, ppis[rng() % 6], waves[rng() % 4])) return 1;
    // the same batch with random groups sharing random prefixes
    const int ng = 1 + int(rng() % 40);
    std::vector<int32_t> group_of(b), group_pages(ng);
    for (auto& g : group_of) g = int32_t(rng() % (ng + 1)) - 1;
    for (auto& g : group_pages) g = int32_t(rng() % 200);
    if (check(lens, hkv, ppis[rng() % 6], waves[rng() % 4], &group_of,
              &group_pages))
      return 1;
  }
  // argument errors must not touch the output or leak
  laminar_plan* p = reinterpret_cast<laminar_plan*>(0x1);
  if (laminar_plan_create(nullptr, nullptr, 256, &p) != LAMINAR_ERR_INVALID_ARG ||
      p != nullptr)
    return fail("null desc");
  laminar_plan_destroy(nullptr);
  std::printf("plan_check OK\n");
  return 0;
}
