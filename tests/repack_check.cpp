// Builds with g++ alone (no HIP): exercises the host halves of repacking
// (laminar_repack_plan, laminar_migration_pairs) and the roofline bound over
// random and edge-case inputs, checking every returned index and count.
// Run under AddressSanitizer and UndefinedBehaviorSanitizer by the tests.
#include <cstdint>
#include <cstdio>
#include <random>
#include <set>
#include <vector>

#include "laminar_repack.h"

static int fail(const char* what) {
  std::printf("FAIL %s\n", what);
  return 1;
}

static int check_plan(std::mt19937& rng, int n) {
  std::vector<laminar_rollout_state> r(size_t(n > 0 ? n : 1));
  std::uniform_int_distribution<int64_t> kv(0, 5000);
  std::uniform_int_distribution<int32_t> reqs(0, 64);
  for (int i = 0; i < n; ++i) {
    r[size_t(i)].kv_used = kv(rng);
    r[size_t(i)].kv_prev = kv(rng);
    r[size_t(i)].num_reqs = reqs(rng);
    r[size_t(i)].reserved = 0;
  }
  std::vector<int32_t> src(size_t(n > 0 ? n : 1), -7), dst(src);
  int32_t np = -1;
  const int64_t kv_max = 1 + kv(rng);
  const int32_t b_max = 1 + reqs(rng);
  if (laminar_repack_plan(r.data(), n, kv_max, b_max, src.data(), dst.data(),
                          &np) != LAMINAR_OK)
    return fail("repack status");
  if (np < 0 || np > n) return fail("repack count");
  for (int i = 0; i < np; ++i)
    if (src[size_t(i)] < 0 || src[size_t(i)] >= n || dst[size_t(i)] < 0 ||
        dst[size_t(i)] >= n || src[size_t(i)] == dst[size_t(i)])
      return fail("repack pair");
  return 0;
}

static int check_pairs(std::mt19937& rng) {
  std::uniform_int_distribution<int> nt(0, 12), len(0, 200), pool(1, 400);
  const int n = nt(rng), sw = 14, dw = 16, src_pages = pool(rng);
  std::vector<int32_t> lens(size_t(n) + 1), table(size_t(n * sw) + 1, -1);
  std::uniform_int_distribution<int> page(0, src_pages - 1);
  int need = 0;
  for (int t = 0; t < n; ++t) {
    lens[size_t(t)] = len(rng);
    const int blocks = (lens[size_t(t)] + 15) / 16;
    for (int j = 0; j < blocks; ++j)
      table[size_t(t * sw + j)] = (t > 0 && j < 2) ? table[size_t(j)] : page(rng);
    need += blocks;
  }
  std::vector<int32_t> free_pages(size_t(need) + 8);
  for (size_t i = 0; i < free_pages.size(); ++i) free_pages[i] = int32_t(1000 + i);
  std::uniform_int_distribution<int> cap_extra(-2, 2);
  const int cap = std::max(0, need + cap_extra(rng));
  std::vector<int32_t> dst(size_t(n * dw) + 1, -9), pairs(size_t(2 * cap) + 2, -9);
  int32_t np = -1, used = -1;
  const laminar_status st = laminar_migration_pairs(
      table.data(), lens.data(), n, sw, free_pages.data(),
      int32_t(free_pages.size()), dst.data(), dw, pairs.data(), cap, &np, &used);
  if (st == LAMINAR_ERR_INVALID_ARG) return 0;   // capacity below the need
  if (st != LAMINAR_OK) return fail("pairs status");
  if (np < 0 || np > cap || used != np) return fail("pairs count");
  std::set<int32_t> dsts;
  for (int i = 0; i < np; ++i) {
    if (pairs[size_t(2 * i)] < 0 || pairs[size_t(2 * i)] >= src_pages)
      return fail("pair source");
    if (!dsts.insert(pairs[size_t(2 * i + 1)]).second) return fail("pair dest");
  }
  for (int t = 0; t < n; ++t) {
    const int blocks = (lens[size_t(t)] + 15) / 16;
    for (int j = 0; j < dw; ++j) {
      const int32_t v = dst[size_t(t * dw + j)];
      if (j < blocks ? dsts.count(v) == 0 : v != -1) return fail("dest row");
    }
  }
  return 0;
}

static int check_roofline(std::mt19937& rng) {
  std::uniform_int_distribution<int32_t> s(1, 1 << 16);
  laminar_model_shape m = {s(rng) % 256 + 1, s(rng), s(rng) % 128 + 1, 1,
                           s(rng) % 512 + 1, s(rng), s(rng) * 16, 2, 2, 2};
  m.kv_heads = 1 + m.q_heads / 8;
  int32_t bound = -1;
  if (laminar_roofline_batch_bound(&m, 2500000000000000ull, 8000000000000ull,
                                   &bound) != LAMINAR_OK || bound < 0)
    return fail("bound");
  double sec = -1.0;
  if (laminar_roofline_step_seconds(&m, s(rng), s(rng), 2500000000000000ull,
                                    8000000000000ull, &sec) != LAMINAR_OK ||
      !(sec > 0.0))
    return fail("step seconds");
  return 0;
}

int main() {
  std::mt19937 rng(7);
  for (int n : {0, 1, 2, 3, 17, 64})
    for (int rep = 0; rep < 40; ++rep)
      if (check_plan(rng, n)) return 1;
  for (int rep = 0; rep < 400; ++rep)
    if (check_pairs(rng)) return 1;
  for (int rep = 0; rep < 400; ++rep)
    if (check_roofline(rng)) return 1;
  int32_t np = 0;
  if (laminar_repack_plan(nullptr, 3, 10, 10, nullptr, nullptr, &np) !=
      LAMINAR_ERR_INVALID_ARG)
    return fail("null rollouts");
  if (laminar_roofline_batch_bound(nullptr, 1, 1, &np) != LAMINAR_ERR_INVALID_ARG)
    return fail("null shape");
  std::printf("repack_check OK\n");
  return 0;
}
