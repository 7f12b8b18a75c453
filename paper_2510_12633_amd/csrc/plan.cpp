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
  if (d->input_row_stride != 0 &&
      (int64_t(d->input_row_stride) < int64_t(d->num_q_heads) * d->head_dim ||
       d->input_row_stride % 8 != 0))
    return LAMINAR_ERR_INVALID_ARG;
  if (d->waves_per_item != 0 && d->waves_per_item != 1 &&
      d->waves_per_item != 2 && d->waves_per_item != 4)
    return LAMINAR_ERR_INVALID_ARG;
  if (d->kv_dtype != LAMINAR_KV_BF16 && d->kv_dtype != LAMINAR_KV_FP8_E4M3FN)
    return LAMINAR_ERR_INVALID_ARG;
  if (d->kv_dtype == LAMINAR_KV_FP8_E4M3FN &&
      (!d->k_scale || !d->v_scale ||
       (reinterpret_cast<uintptr_t>(d->k_scale) & 3) != 0 ||
       (reinterpret_cast<uintptr_t>(d->v_scale) & 3) != 0))
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

laminar_status validate_groups(const laminar_attn_desc* d,
                               const int32_t* group_of, int32_t num_groups,
                               const int32_t* group_pages) {
  if (num_groups < 0) return LAMINAR_ERR_INVALID_ARG;
  if (num_groups > 0 && (!group_of || !group_pages))
    return LAMINAR_ERR_INVALID_ARG;
  if (num_groups == 0) return LAMINAR_OK;
  for (int32_t b = 0; b < d->batch; ++b)
    if (group_of[b] < -1 || group_of[b] >= num_groups)
      return LAMINAR_ERR_INVALID_ARG;
  for (int32_t g = 0; g < num_groups; ++g)
    if (group_pages[g] < 0) return LAMINAR_ERR_INVALID_ARG;
  return LAMINAR_OK;
}

// Page-aligned cut of `pages` into n = ceil(pages / cap) pieces (one empty
// piece for 0 pages). Plain: near-equal pieces, the first ones one page
// longer. In halves (n >= 2): the first ceil(n / 2) pieces are twice as
// long as the others, each half near-equal, so a unit's later pieces are
// short ones that can join the dynamic tail.
struct Cut {
  uint32_t n, k;          // pieces; the first k are the long half
  uint32_t lb, lr, sb, sr;  // long: size lb, first lr one longer; short alike
  Cut() : n(1), k(1), lb(0), lr(0), sb(0), sr(0) {}
  Cut(uint32_t pages, uint32_t cap, bool halves = false) {
    n = pages == 0 ? 1 : (pages - 1) / cap + 1;
    k = n;
    lb = pages / n;
    lr = pages - lb * n;
    sb = sr = 0;
    if (halves && n >= 2) {
      const uint32_t kk = (n + 1) / 2;
      // long pieces weigh 2, short ones 1: the long half holds
      // pages * 2 kk / (2 kk + n - kk), rounded
      const uint64_t w = uint64_t(kk) + n;
      const uint32_t lng = uint32_t((uint64_t(pages) * 2 * kk + w / 2) / w);
      const uint32_t sht = pages - lng;
      if (sht / (n - kk) >= 2) {          // short pieces keep a page pair
        k = kk;
        lb = lng / k;
        lr = lng - lb * k;
        sb = sht / (n - k);
        sr = sht - sb * (n - k);
      }
    }
  }
  uint32_t size(uint32_t i) const {
    return i < k ? lb + (i < lr ? 1u : 0u) : sb + (i - k < sr ? 1u : 0u);
  }
};

// One group chunk that is decoded as a cascade: up to waves x (16 / g)
// members whose first `pages` blocks map to the same physical pages.
struct Chunk {
  std::vector<int32_t> members;   // trajectory indices, increasing
  int32_t row;                    // longest member: its table row is read,
                                  // its length bounds every row's tokens
  uint32_t pages;                 // shared pages decoded once
  Cut cut;
};

// XCD-aware launch order. The hardware deals workgroup k to XCD k % 8, and
// each XCD has its own L2. The hkv items of one page range of one
// trajectory (or cascade chunk), one per kv-head, form a group: they read
// the same block-table entries and, for fp8 pools, the same lines of the
// [page][kv-head] scale arrays, and their K and V tiles of a page are
// adjacent in HBM. The list arrives longest first with each group's items
// next to each other; every run of eight groups is laid out kv-head-major,
// item (group x, kv-head h) at run start + 8 h + x, so that a group's items
// sit on one XCD and run there side by side and the shared lines come from
// its L2 instead of once per kv-head from HBM. A last run of fewer than
// eight groups keeps the layout without that property.
void xcd_order(Item* items, int64_t n, int32_t hkv) {
  constexpr int64_t kXcds = 8;
  if (hkv <= 1) return;
  std::vector<Item> run(size_t(kXcds * hkv));
  for (int64_t r = 0; r < n; r += kXcds * hkv) {
    const int64_t len = std::min(n - r, kXcds * hkv);
    const int64_t groups = len / hkv;          // n is a multiple of hkv
    std::copy(items + r, items + r + len, run.begin());
    for (int64_t x = 0; x < groups; ++x)
      for (int64_t h = 0; h < hkv; ++h)
        items[r + h * groups + x] = run[size_t(x * hkv + h)];
  }
}

laminar_status build(const laminar_attn_desc* desc, const int32_t* lens,
                     const int32_t* group_of, int32_t num_groups,
                     const int32_t* group_pages, int32_t num_cus,
                     laminar_plan** out) {
  if (!out) return LAMINAR_ERR_INVALID_ARG;
  *out = nullptr;
  laminar_status st = validate(desc, lens, num_cus);
  if (st != LAMINAR_OK) return st;
  st = validate_groups(desc, group_of, num_groups, group_pages);
  if (st != LAMINAR_OK) return st;

  laminar_plan* p = new (std::nothrow) laminar_plan();
  if (!p) return LAMINAR_ERR_INVALID_ARG;
  try {
  p->desc = *desc;
  const int32_t B = desc->batch, hkv = desc->num_kv_heads;
  p->group = desc->num_q_heads / hkv;
  p->waves = desc->waves_per_item ? desc->waves_per_item
                                  : laminar_detail::kDefaultWaves;
  const int32_t W = p->waves;
  std::vector<uint32_t> pages(static_cast<size_t>(B));
  for (int32_t b = 0; b < B; ++b) pages[size_t(b)] = (uint32_t(lens[b]) + 15) / 16;

  // Cascade chunks. A chunk item gives each of its W wavefronts the rows of
  // 16 / g members and walks every shared page in each wavefront, so one
  // item reads the shared pages once for W * (16 / g) members. Chunks of
  // fewer than two members, or with nothing shared, decode as usual.
  std::vector<Chunk> chunks;
  std::vector<uint32_t> first(static_cast<size_t>(B), 0);   // first own page
  std::vector<int32_t> chunk_of(static_cast<size_t>(B), -1);
  if (num_groups > 0) {
    const int32_t cap = W * (16 / p->group);
    std::vector<std::vector<int32_t>> groups(static_cast<size_t>(num_groups));
    for (int32_t b = 0; b < B; ++b)
      if (group_of[b] >= 0) groups[size_t(group_of[b])].push_back(b);
    for (int32_t g = 0; g < num_groups; ++g) {
      const auto& m = groups[size_t(g)];
      for (size_t s = 0; s < m.size(); s += size_t(cap)) {
        Chunk c;
        c.members.assign(m.begin() + long(s),
                         m.begin() + long(std::min(m.size(), s + size_t(cap))));
        // the member with the most tokens: its length bounds the valid
        // slots of every shared page, for all rows
        c.row = c.members[0];
        for (int32_t b : c.members)
          if (lens[b] > lens[c.row]) c.row = b;
        c.pages = std::min(uint32_t(group_pages[g]), pages[size_t(c.row)]);
        if (c.members.size() < 2 || c.pages == 0) continue;
        for (int32_t b : c.members) {
          first[size_t(b)] = std::min(pages[size_t(b)], c.pages);
          chunk_of[size_t(b)] = int32_t(chunks.size());
        }
        chunks.push_back(std::move(c));
      }
    }
  }

  // Split size. Work is counted in wavefront-time: a page of an ordinary
  // item costs 1 (its W wavefronts share the pages), a page of a cascade
  // item costs W (each wavefront walks it for its own rows).
  int64_t work = 0;
  for (int32_t b = 0; b < B; ++b) work += int64_t(pages[size_t(b)] - first[size_t(b)]) * hkv;
  for (const Chunk& c : chunks) work += int64_t(c.pages) * hkv * W;
  const int64_t resident = int64_t(num_cus) *
      std::max(1, laminar_detail::kResidentWavesPerCU / W);
  const int64_t step = 2 * int64_t(W);          // one page pair per wave
  // Aim for num / den items per resident workgroup; every wave of an item
  // gets at least one pair of pages.
  auto chunk_for = [&](int64_t num, int64_t den) {
    const int64_t target = resident * num / den;
    const int64_t c = std::max<int64_t>(step, (work + target - 1) / target);
    return (c + step - 1) / step * step;
  };
  int64_t chunk;
  bool halves = false;
  if (desc->pages_per_item > 0) {
    chunk = desc->pages_per_item;
  } else {
    chunk = chunk_for(laminar_detail::kItemsPerSlotNum,
                      laminar_detail::kItemsPerSlotDen);
    // A batch that mixes units shorter than half a piece (whole items that
    // fall to the dynamic tail) with units cut into several pieces aims
    // for kMixedItemsPerSlot items per slot and cuts the long units in
    // halves, so their short second halves join the tail too: measured
    // 4% faster on the TP-4 share of the 32B workload, 0.6% on
    // 7b_pre_repack and 0.2% on the 32B workload. A batch of long units
    // only (post_repack) keeps equal pieces and no tail, which halves made
    // 3-7% slower, and so do cascade plans, which have no dynamic tail
    // (halves made the agentic mixes 0.5-1% slower). Nor do batches with
    // more than 4 kv-heads: the kv-heads of a page share its fp8 scale and
    // block-table lines, which the XCD-grouped order keeps in one L2, and
    // the dynamic tail hands its items to any XCD (the 32B workload, 8
    // kv-heads: 1.017 x the algorithmic HBM bytes with halves, 1.010
    // without, for 0.2% of time).
    bool has_short = false, has_long = false;
    for (int32_t b = 0; b < B && chunks.empty(); ++b) {
      const int64_t own = int64_t(pages[size_t(b)]) - first[size_t(b)];
      has_short |= own > 0 && 2 * own < chunk;
      has_long |= own > chunk;
    }
    if (has_short && has_long && hkv <= 4) {
      halves = true;
      chunk = chunk_for(laminar_detail::kMixedItemsPerSlot, 1);
    }
  }
  const uint32_t chunk32 = uint32_t(std::min<int64_t>(chunk, UINT32_MAX));
  // cascade pieces: the same wavefront-time, whole page pairs
  const uint32_t cchunk =
      std::max<uint32_t>(2, uint32_t(std::min<int64_t>(chunk / W, UINT32_MAX)) & ~1u);
  for (Chunk& c : chunks) c.cut = Cut(c.pages, cchunk);

  std::vector<Cut> cuts(static_cast<size_t>(B));
  int64_t total = 0, merges = 0, slots = 0, members = 0;
  uint32_t longest = 0;                          // longest item, wave-time
  uint32_t max_piece = 0;                        // longest ordinary item
  for (int32_t b = 0; b < B; ++b) {
    const uint32_t own = pages[size_t(b)] - first[size_t(b)];
    const bool cas = chunk_of[size_t(b)] >= 0;
    // a cascade member with nothing of its own has no ordinary item
    Cut c = (cas && own == 0) ? Cut() : Cut(own, chunk32, halves);
    if (cas && own == 0) c.n = 0;
    cuts[size_t(b)] = c;
    total += int64_t(c.n) * hkv;
    if (c.n) {
      longest = std::max(longest, c.size(0));
      max_piece = std::max(max_piece, c.size(0));
    }
    const int64_t n_all = c.n + (cas ? chunks[size_t(chunk_of[size_t(b)])].cut.n : 0);
    if (cas || n_all > 1) {
      merges += hkv;
      slots += n_all * hkv;
    }
  }
  // the bound the pieces respect: the split size, or the long half's pieces
  p->pages_per_item = int32_t(
      std::min<int64_t>(std::max<int64_t>(chunk, max_piece), INT32_MAX));
  for (const Chunk& c : chunks) {
    total += int64_t(c.cut.n) * hkv;
    longest = std::max<uint32_t>(longest, uint32_t(W) * c.cut.size(0));
    members += int64_t(c.members.size()) * hkv;
  }
  if (total > INT32_MAX || slots > INT32_MAX || members > INT32_MAX)
    throw std::length_error("items");

  p->num_items = int32_t(total);
  p->num_merges = int32_t(merges);
  p->num_slots = int32_t(slots);
  p->num_cascade_units = int32_t(chunks.size()) * hkv;
  p->num_cascade_members = int32_t(members);
  size_t off = 0;
  p->off_items = off;
  off = align256(off + size_t(total) * 16);
  p->off_merges = off;
  off = align256(off + size_t(merges) * 16);
  p->off_cunits = off;
  off = align256(off + size_t(p->num_cascade_units) * 16);
  p->off_cmembers = off;
  off = align256(off + size_t(members) * 8);
  p->off_tail = off;
  off = align256(off + sizeof(int32_t));
  p->off_lse = off;
  off = align256(off + size_t(slots) * p->group * sizeof(float));
  p->off_o = off;
  off = align256(off + size_t(slots) * p->group * desc->head_dim * sizeof(float));
  p->ws_bytes = off;

  // The tables are built in place in the byte image of the workspace up to
  // the partial results.
  p->tables.assign(p->off_lse / sizeof(int32_t), 0);
  Item* items = reinterpret_cast<Item*>(p->tables.data() + p->off_items / 4);
  Item* mrec = reinterpret_cast<Item*>(p->tables.data() + p->off_merges / 4);
  Item* cunit = reinterpret_cast<Item*>(p->tables.data() + p->off_cunits / 4);
  int32_t* cmem = p->tables.data() + p->off_cmembers / 4;

  // Launch order: longest (in wavefront-time) first; equal lengths keep
  // (cascade units, then trajectory, kv-head, page) order. The hardware
  // dispatcher hands the workgroups to CUs greedily as earlier ones finish.
  // A stable counting sort on the length.
  std::vector<int64_t> start(size_t(longest) + 2, 0);
  for (const Chunk& c : chunks)
    for (uint32_t i = 0; i < c.cut.n; ++i) start[longest - W * c.cut.size(i)] += hkv;
  for (const Cut& c : cuts)
    for (uint32_t i = 0; i < c.n; ++i) start[longest - c.size(i)] += hkv;
  int64_t acc = 0;
  for (auto& v : start) { const int64_t c = v; v = acc; acc += c; }

  // Slots: every unit of a cascade member, and every other unit cut into
  // several pieces, gets consecutive partial slots (cascade pieces first,
  // then its own pieces in page order) and one merge record.
  std::vector<int32_t> slot0(size_t(B) * hkv, -1);
  int32_t next_slot = 0, m = 0;
  for (int64_t u = 0; u < int64_t(B) * hkv; ++u) {
    const int32_t b = int32_t(u / hkv);
    const int32_t ci = chunk_of[size_t(b)];
    const int32_t n_all = int32_t(cuts[size_t(b)].n) +
                          (ci >= 0 ? int32_t(chunks[size_t(ci)].cut.n) : 0);
    if (ci >= 0 || n_all > 1) {
      slot0[size_t(u)] = next_slot;
      mrec[m++] = {int32_t(u), next_slot, n_all, 0};
      next_slot += n_all;
    }
  }
  // Items. The kv-heads of a unit are cut alike, so the hkv items of one
  // page range (a group) have one size; they are placed next to each other
  // (trajectory, piece, kv-head order), which xcd_order relies on.
  for (int32_t b = 0; b < B; ++b) {
    const Cut& c = cuts[size_t(b)];
    const int32_t ci = chunk_of[size_t(b)];
    const uint32_t ncas = ci >= 0 ? chunks[size_t(ci)].cut.n : 0;
    int32_t pos = int32_t(first[size_t(b)]);
    for (uint32_t i = 0; i < c.n; ++i) {
      const uint32_t sz = c.size(i);
      for (int32_t h = 0; h < hkv; ++h) {
        const int64_t u = int64_t(b) * hkv + h;
        const int32_t s0 = slot0[size_t(u)];
        items[start[longest - sz]++] = {int32_t(u), pos, pos + int32_t(sz),
                                        s0 >= 0 ? s0 + int32_t(ncas + i) : -1};
      }
      pos += int32_t(sz);
    }
  }
  // Cascade units (chunk, kv-head): header (row, members, first member
  // record, kv-head) and member records (trajectory, first slot); then
  // their items, again a group of hkv items per piece.
  int32_t mo = 0;
  for (size_t ci = 0; ci < chunks.size(); ++ci) {
    const Chunk& c = chunks[ci];
    for (int32_t h = 0; h < hkv; ++h) {
      const int32_t cu = int32_t(ci) * hkv + h;
      cunit[cu] = {c.row, int32_t(c.members.size()), mo, h};
      for (int32_t b : c.members) {
        cmem[2 * mo] = b;
        cmem[2 * mo + 1] = slot0[size_t(b) * hkv + h];
        ++mo;
      }
    }
    int32_t pos = 0;
    for (uint32_t i = 0; i < c.cut.n; ++i) {
      const uint32_t sz = c.cut.size(i);
      for (int32_t h = 0; h < hkv; ++h) {
        const int32_t cu = int32_t(ci) * hkv + h;
        items[start[longest - W * sz]++] = {-(cu + 1), pos, pos + int32_t(sz),
                                            int32_t(i)};
      }
      pos += int32_t(sz);
    }
  }
  xcd_order(items, total, hkv);
  // Dynamic tail. Workgroups are dealt to the eight XCDs round-robin by
  // index and the XCDs stream at rates up to ~10% apart, so a fixed
  // assignment ends when the slowest XCD ends. The smallest items (at most
  // half the size of the largest, together at most half the work) are
  // therefore not bound to an index: each workgroup past num_main takes
  // the next of them from a counter when the hardware starts it, so XCDs
  // that run ahead take more of the tail. Plans with cascade items, or
  // whose items are all about equal (nothing to rebalance, only the
  // counter's latency to pay), keep every item bound to its index.
  p->num_main = int32_t(total);
  if (chunks.empty() && total > 0) {
    int64_t all = 0;
    for (int64_t i = 0; i < total; ++i) all += items[i].p1 - items[i].p0;
    const int32_t small = (items[0].p1 - items[0].p0) / 2;
    int64_t acc = 0, i = total;
    while (i > 0) {
      const int32_t sz = items[i - 1].p1 - items[i - 1].p0;
      if (sz > small || 2 * (acc + sz) > all) break;
      acc += sz;
      --i;
    }
    p->num_main = int32_t(i);
  }
  } catch (...) {     // host allocation failure or too many items: report
    delete p;
    return LAMINAR_ERR_INVALID_ARG;
  }
  *out = p;
  return LAMINAR_OK;
}

}  // namespace

extern "C" {

laminar_status laminar_plan_create(const laminar_attn_desc* desc,
                                   const int32_t* seq_lens_host,
                                   int32_t num_cus, laminar_plan** out) {
  return build(desc, seq_lens_host, nullptr, 0, nullptr, num_cus, out);
}

laminar_status laminar_plan_create_cascade(const laminar_attn_desc* desc,
                                           const int32_t* seq_lens_host,
                                           const int32_t* group_of_host,
                                           int32_t num_groups,
                                           const int32_t* group_pages_host,
                                           int32_t num_cus, laminar_plan** out) {
  return build(desc, seq_lens_host, group_of_host, num_groups,
               group_pages_host, num_cus, out);
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

int32_t laminar_plan_num_dynamic_items(const laminar_plan* plan) {
  return plan ? plan->num_items - plan->num_main : -1;
}

int32_t laminar_plan_num_cascade_units(const laminar_plan* plan) {
  return plan ? plan->num_cascade_units : -1;
}

int32_t laminar_plan_num_cascade_members(const laminar_plan* plan) {
  return plan ? plan->num_cascade_members : -1;
}

int32_t laminar_plan_cascade_units_copy(const laminar_plan* plan, int32_t* dst,
                                        int32_t capacity) {
  if (!plan || !dst || capacity < 0) return -1;
  const int32_t n = std::min(capacity, plan->num_cascade_units);
  std::memcpy(dst, plan->tables.data() + plan->off_cunits / 4, size_t(n) * 16);
  return n;
}

int32_t laminar_plan_cascade_members_copy(const laminar_plan* plan,
                                          int32_t* dst, int32_t capacity) {
  if (!plan || !dst || capacity < 0) return -1;
  const int32_t n = std::min(capacity, plan->num_cascade_members);
  std::memcpy(dst, plan->tables.data() + plan->off_cmembers / 4, size_t(n) * 8);
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
