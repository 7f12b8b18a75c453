// Host planner for split-KV paged decode attention.
//
// The paper's repack consolidates long-tail trajectories onto a few rollouts
// (§5.2) so that one decode batch holds a handful of very long trajectories
// next to many short ones. One GPU must still keep all its CUs busy on such a
// batch, so the planner cuts every (trajectory, kv-head) unit of
// ceil(n/16) pages into near-equal page-aligned ranges and orders the work
// longest first; ranges of a unit that was cut are later combined by the
// log-sum-exp merge. Pure host C++: no HIP call, no device memory.

#include <algorithm>
#include <cstring>
#include <functional>
#include <new>
#include <numeric>
#include <utility>

#include "plan_internal.h"

namespace {

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

struct Piece { int32_t unit, p0, p1; };
struct Item { int32_t unit, p0, p1, slot; };

laminar_status validate(const laminar_attn_desc* d, const int32_t* lens,
                        int32_t num_cus) {
  if (!d || num_cus <= 0) return LAMINAR_ERR_INVALID_ARG;
  if (d->batch < 0 || d->num_q_heads <= 0 || d->num_kv_heads <= 0 ||
      d->num_pages <= 0 || d->max_blocks_per_seq < 0 || d->head_dim <= 0)
    return LAMINAR_ERR_INVALID_ARG;
  if (d->batch > 0 && !lens) return LAMINAR_ERR_INVALID_ARG;
  if (d->num_q_heads % d->num_kv_heads != 0) return LAMINAR_ERR_INVALID_ARG;
  if (!(d->softmax_scale > 0.0f)) return LAMINAR_ERR_INVALID_ARG;
  if (d->pages_per_item < 0) return LAMINAR_ERR_INVALID_ARG;
  if (d->waves_per_item != 0 && d->waves_per_item != 1 &&
      d->waves_per_item != 2 && d->waves_per_item != 4)
    return LAMINAR_ERR_INVALID_ARG;
  if (d->kv_dtype != LAMINAR_KV_BF16 && d->kv_dtype != LAMINAR_KV_FP8_E4M3FN)
    return LAMINAR_ERR_INVALID_ARG;
  if (d->kv_dtype == LAMINAR_KV_FP8_E4M3FN && (!d->k_scale || !d->v_scale))
    return LAMINAR_ERR_INVALID_ARG;
  if (d->page_size != 16) return LAMINAR_ERR_UNSUPPORTED;
  if (d->head_dim != 64 && d->head_dim != 128) return LAMINAR_ERR_UNSUPPORTED;
  if (d->num_q_heads / d->num_kv_heads > 16) return LAMINAR_ERR_UNSUPPORTED;
  for (int32_t b = 0; b < d->batch; ++b) {
    if (lens[b] < 0) return LAMINAR_ERR_INVALID_ARG;
    const int64_t pages = (int64_t(lens[b]) + 15) / 16;
    if (pages > d->max_blocks_per_seq) return LAMINAR_ERR_INVALID_ARG;
  }
  return LAMINAR_OK;
}

}  // namespace

extern "C" {

laminar_status laminar_plan_create(const laminar_attn_desc* desc,
                                   const int32_t* seq_lens_host,
                                   int32_t num_cus, laminar_plan** out) {
  if (!out) return LAMINAR_ERR_INVALID_ARG;
  *out = nullptr;
  laminar_status st = validate(desc, seq_lens_host, num_cus);
  if (st != LAMINAR_OK) return st;

  laminar_plan* p = new (std::nothrow) laminar_plan();
  if (!p) return LAMINAR_ERR_INVALID_ARG;
  try {
  p->desc = *desc;
  const int32_t B = desc->batch, hkv = desc->num_kv_heads;
  p->group = desc->num_q_heads / hkv;
  p->waves = desc->waves_per_item ? desc->waves_per_item
                                  : laminar_detail::kDefaultWaves;
  const int64_t units = int64_t(B) * hkv;
  std::vector<int64_t> upages(static_cast<size_t>(units), 0);
  int64_t work = 0;                        // (page, kv-head) tiles
  for (int32_t b = 0; b < B; ++b)
    for (int32_t h = 0; h < hkv; ++h) {
      upages[size_t(b) * hkv + h] = (int64_t(seq_lens_host[b]) + 15) / 16;
      work += upages[size_t(b) * hkv + h];
    }
  const int64_t resident = int64_t(num_cus) *
      std::max(1, laminar_detail::kResidentWavesPerCU / p->waves);
  const int64_t step = 2 * int64_t(p->waves);   // one page pair per wave

  int64_t chunk;
  if (desc->pages_per_item > 0) {
    chunk = desc->pages_per_item;
  } else {
    // Aim for kItemsPerSlot items per resident workgroup; every wave of an
    // item gets at least one pair of pages.
    const int64_t target = resident * laminar_detail::kItemsPerSlotNum /
                           laminar_detail::kItemsPerSlotDen;
    chunk = std::max<int64_t>(step, (work + target - 1) / target);
    chunk = (chunk + step - 1) / step * step;
  }
  p->pages_per_item = int32_t(std::min<int64_t>(chunk, INT32_MAX));

  // Near-equal page-aligned pieces of every unit, launched longest first
  // (ties keep trajectory, kv-head, page order); the hardware dispatcher
  // hands them to CUs greedily as workgroups finish.
  std::vector<Piece> order;
  order.reserve(size_t(units) + size_t(work / chunk) + 1);
  for (int64_t u = 0; u < units; ++u) {
    const int64_t pages = upages[size_t(u)];
    const int64_t n = pages == 0 ? 1 : (pages + chunk - 1) / chunk;
    const int64_t base = pages / n, rem = pages % n;
    int64_t pos = 0;
    for (int64_t i = 0; i < n; ++i) {
      const int64_t sz = base + (i < rem ? 1 : 0);
      order.push_back({int32_t(u), int32_t(pos), int32_t(pos + sz)});
      pos += sz;
    }
  }
  std::stable_sort(order.begin(), order.end(),
                   [](const Piece& a, const Piece& b) {
                     return (a.p1 - a.p0) > (b.p1 - b.p0);
                   });

  // Partial slots: a unit cut into several pieces gets consecutive slots in
  // page order and one merge record; a unit in one piece writes directly.
  std::vector<int32_t> count(static_cast<size_t>(units), 0);
  std::vector<int32_t> first_slot(static_cast<size_t>(units), -1);
  for (const Piece& pc : order) ++count[size_t(pc.unit)];
  std::vector<Item> merges;            // (unit, slot0, n, 0)
  int32_t slots = 0;
  for (int64_t u = 0; u < units; ++u)
    if (count[size_t(u)] > 1) {
      first_slot[size_t(u)] = slots;
      merges.push_back({int32_t(u), slots, count[size_t(u)], 0});
      slots += count[size_t(u)];
    }
  // Rank of each piece among its unit's pieces by first page.
  std::vector<Item> items(order.size());
  {
    std::vector<std::vector<std::pair<int32_t, int32_t>>> per_unit;
    std::vector<int32_t> split_index(static_cast<size_t>(units), -1);
    for (size_t i = 0; i < order.size(); ++i) {
      const Piece& pc = order[i];
      items[i] = {pc.unit, pc.p0, pc.p1, -1};
      if (count[size_t(pc.unit)] > 1) {
        int32_t& si = split_index[size_t(pc.unit)];
        if (si < 0) {
          si = int32_t(per_unit.size());
          per_unit.emplace_back();
        }
        per_unit[size_t(si)].push_back({pc.p0, int32_t(i)});
      }
    }
    for (auto& v : per_unit) {
      std::sort(v.begin(), v.end());
      const int32_t unit = items[size_t(v[0].second)].unit;
      for (size_t r = 0; r < v.size(); ++r)
        items[size_t(v[r].second)].slot = first_slot[size_t(unit)] + int32_t(r);
    }
  }

  p->num_items = int32_t(items.size());
  p->num_merges = int32_t(merges.size());
  p->num_slots = slots;

  size_t off = 0;
  p->off_items = off;
  off = align256(off + items.size() * 16);
  p->off_merges = off;
  off = align256(off + merges.size() * 16);
  p->off_lse = off;
  off = align256(off + size_t(slots) * p->group * sizeof(float));
  p->off_o = off;
  off = align256(off + size_t(slots) * p->group * desc->head_dim * sizeof(float));
  p->ws_bytes = off;

  // Byte image of the workspace up to the partial results: items, then
  // merges, at their section offsets (zero padding between).
  p->tables.assign(p->off_lse / sizeof(int32_t), 0);
  if (!items.empty())
    std::memcpy(p->tables.data() + p->off_items / 4, items.data(),
                items.size() * sizeof(Item));
  if (!merges.empty())
    std::memcpy(p->tables.data() + p->off_merges / 4, merges.data(),
                merges.size() * sizeof(Item));
  } catch (...) {            // host allocation failure: report, never throw
    delete p;
    return LAMINAR_ERR_INVALID_ARG;
  }
  *out = p;
  return LAMINAR_OK;
}

size_t laminar_plan_workspace_bytes(const laminar_plan* plan) {
  return plan ? plan->ws_bytes : 0;
}

int32_t laminar_plan_num_items(const laminar_plan* plan) {
  return plan ? plan->num_items : -1;
}

int32_t laminar_plan_num_merges(const laminar_plan* plan) {
  return plan ? plan->num_merges : -1;
}

int32_t laminar_plan_pages_per_item(const laminar_plan* plan) {
  return plan ? plan->pages_per_item : -1;
}

int32_t laminar_plan_waves_per_item(const laminar_plan* plan) {
  return plan ? plan->waves : -1;
}

int32_t laminar_plan_items_copy(const laminar_plan* plan, int32_t* dst,
                                int32_t capacity) {
  if (!plan || !dst || capacity < 0) return -1;
  const int32_t n = std::min(capacity, plan->num_items);
  std::memcpy(dst, plan->tables.data() + plan->off_items / 4, size_t(n) * 16);
  return n;
}

int32_t laminar_plan_merges_copy(const laminar_plan* plan, int32_t* dst,
                                 int32_t capacity) {
  if (!plan || !dst || capacity < 0) return -1;
  const int32_t n = std::min(capacity, plan->num_merges);
  std::memcpy(dst, plan->tables.data() + plan->off_merges / 4, size_t(n) * 16);
  return n;
}

void laminar_plan_destroy(laminar_plan* plan) { delete plan; }

const char* laminar_status_string(laminar_status s) {
  switch (s) {
    case LAMINAR_OK: return "ok";
    case LAMINAR_ERR_INVALID_ARG: return "invalid argument";
    case LAMINAR_ERR_UNSUPPORTED: return "unsupported configuration";
    case LAMINAR_ERR_WORKSPACE: return "workspace missing, too small or misaligned";
    case LAMINAR_ERR_HIP: return "HIP runtime error";
  }
  return "unknown status";
}

}  // extern "C"
