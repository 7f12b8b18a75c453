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
#include <new>
#include <stdexcept>

#include "plan_internal.h"

namespace {

size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

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
  int64_t work = 0;                        // (page, kv-head) tiles
  for (int32_t b = 0; b < B; ++b)
    work += (int64_t(seq_lens_host[b]) + 15) / 16 * hkv;
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

  // Near-equal page-aligned pieces of every unit (trajectory, kv-head):
  // n = ceil(pages / chunk) pieces, the first pages % n of them one page
  // longer; all kv-heads of a trajectory are cut alike. A unit cut into
  // several pieces gets n consecutive partial slots in page order and one
  // merge record; a unit in one piece writes out/lse directly.
  struct Cut { uint32_t n, base, rem; };
  std::vector<Cut> cuts(static_cast<size_t>(B));
  const uint32_t chunk32 = uint32_t(std::min<int64_t>(chunk, UINT32_MAX));
  int64_t total = 0, merges = 0, slots = 0;
  uint32_t longest = 0;
  for (int32_t b = 0; b < B; ++b) {
    const uint32_t pages = (uint32_t(seq_lens_host[b]) + 15) / 16;  // < 2^27
    const uint32_t n = pages == 0 ? 1 : (pages - 1) / chunk32 + 1;
    const uint32_t base = pages / n;
    const uint32_t rem = pages - base * n;
    cuts[size_t(b)] = {n, base, rem};
    total += int64_t(n) * hkv;
    longest = std::max(longest, base + (rem ? 1 : 0));
    if (n > 1) {
      merges += hkv;
      slots += int64_t(n) * hkv;
    }
  }
  if (total > INT32_MAX || slots > INT32_MAX) throw std::length_error("items");

  p->num_items = int32_t(total);
  p->num_merges = int32_t(merges);
  p->num_slots = int32_t(slots);
  size_t off = 0;
  p->off_items = off;
  off = align256(off + size_t(total) * 16);
  p->off_merges = off;
  off = align256(off + size_t(merges) * 16);
  p->off_lse = off;
  off = align256(off + size_t(slots) * p->group * sizeof(float));
  p->off_o = off;
  off = align256(off + size_t(slots) * p->group * desc->head_dim * sizeof(float));
  p->ws_bytes = off;

  // The tables are built in place in the byte image of the workspace up to
  // the partial results (items, then merges, at their section offsets).
  p->tables.assign(p->off_lse / sizeof(int32_t), 0);
  Item* items = reinterpret_cast<Item*>(p->tables.data() + p->off_items / 4);
  Item* mrec = reinterpret_cast<Item*>(p->tables.data() + p->off_merges / 4);

  // Launch order: longest first; equal lengths keep (trajectory, kv-head,
  // page) order. The hardware dispatcher hands the workgroups to CUs
  // greedily as earlier ones finish. A stable counting sort on the length.
  std::vector<int64_t> start(size_t(longest) + 2, 0);
  for (const Cut& c : cuts) {
    start[longest - c.base] += int64_t(c.n - c.rem) * hkv;
    if (c.rem) start[longest - c.base - 1] += int64_t(c.rem) * hkv;
  }
  int64_t acc = 0;
  for (auto& v : start) { const int64_t c = v; v = acc; acc += c; }
  int32_t next_slot = 0, m = 0;
  for (int64_t u = 0; u < int64_t(B) * hkv; ++u) {
    const Cut c = cuts[size_t(u / hkv)];
    const bool split = c.n > 1;
    if (split) mrec[m++] = {int32_t(u), next_slot, int32_t(c.n), 0};
    int32_t pos = 0;
    for (uint32_t i = 0; i < c.n; ++i) {
      const uint32_t sz = c.base + (i < c.rem ? 1 : 0);
      items[start[longest - sz]++] = {int32_t(u), pos, pos + int32_t(sz),
                                      split ? next_slot + int32_t(i) : -1};
      pos += int32_t(sz);
    }
    if (split) next_slot += int32_t(c.n);
  }
  } catch (...) {     // host allocation failure or too many items: report
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
