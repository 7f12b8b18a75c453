// Trajectory repacking, host side: the best-fit consolidation plan, the
// page assignment of a migration, and the roofline batch bound B that the
// plan takes as input. Pure host C++: no HIP call.
//
// The plan follows the paper's Algorithm 1 (§5.2): candidates are the
// rollouts whose KV usage is falling and below the limit and that run fewer
// trajectories than the roofline batch bound; they are visited from the
// least used up, and each that has neither been emptied nor received
// trajectories moves into the candidate that can take it and ends up
// fullest. Loads planned into each candidate are kept incrementally, so a
// visit costs one pass over the candidates.

#include <algorithm>
#include <cstring>
#include <numeric>
#include <unordered_map>
#include <vector>

#include "laminar_repack.h"

namespace {

bool shape_ok(const laminar_model_shape* m) {
  return m && m->layers > 0 && m->hidden > 0 && m->q_heads > 0 &&
         m->kv_heads > 0 && m->head_dim > 0 && m->intermediate > 0 &&
         m->vocab > 0 && m->weight_bytes > 0 && m->act_bytes >= 0 &&
         m->kv_bytes > 0;
}

// (K, N) of every projection of one decode step; calls f(K, N).
template <class F>
void for_each_projection(const laminar_model_shape* m, F f) {
  const int64_t h = m->hidden, d = m->head_dim;
  for (int32_t l = 0; l < m->layers; ++l) {
    f(h, (int64_t(m->q_heads) + 2 * m->kv_heads) * d);
    f(int64_t(m->q_heads) * d, h);
    f(h, 2 * int64_t(m->intermediate));
    f(int64_t(m->intermediate), h);
  }
  f(h, int64_t(m->vocab));
}

}  // namespace

extern "C" {

laminar_status laminar_repack_plan(const laminar_rollout_state* r, int32_t n,
                                   int64_t kv_max, int32_t batch_max,
                                   int32_t* src_out, int32_t* dst_out,
                                   int32_t* num_pairs) {
  if (!num_pairs || n < 0 || kv_max < 0 || batch_max < 0)
    return LAMINAR_ERR_INVALID_ARG;
  *num_pairs = 0;
  if (n > 0 && (!r || !src_out || !dst_out)) return LAMINAR_ERR_INVALID_ARG;
  for (int32_t i = 0; i < n; ++i)
    if (r[i].kv_used < 0 || r[i].kv_prev < 0 || r[i].num_reqs < 0)
      return LAMINAR_ERR_INVALID_ARG;
  try {
    std::vector<int32_t> s;                         // candidates
    for (int32_t i = 0; i < n; ++i)
      if (r[i].kv_used < std::min(kv_max, r[i].kv_prev) &&
          r[i].num_reqs < batch_max)
        s.push_back(i);
    std::stable_sort(s.begin(), s.end(), [&](int32_t a, int32_t b) {
      return r[a].kv_used < r[b].kv_used;
    });
    const size_t m = s.size();
    // usage and trajectories of each candidate including what is planned
    // into it; flags: emptied (moved away) and received (kept)
    std::vector<int64_t> load(m), reqs(m);
    std::vector<char> emptied(m, 0), received(m, 0);
    for (size_t i = 0; i < m; ++i) {
      load[i] = r[s[i]].kv_used;
      reqs[i] = r[s[i]].num_reqs;
    }
    int32_t k = 0;
    for (size_t i = 0; i < m; ++i) {
      if (emptied[i] || received[i]) continue;
      const int64_t cu = r[s[i]].kv_used, nu = r[s[i]].num_reqs;
      int64_t best = -1;
      size_t pick = m;
      for (size_t j = 0; j < m; ++j) {
        if (j == i || emptied[j]) continue;
        if (load[j] + cu > kv_max || reqs[j] + nu > batch_max) continue;
        if (load[j] > best) {           // first of equally full ones wins
          best = load[j];
          pick = j;
        }
      }
      if (pick == m) continue;
      load[pick] += cu;
      reqs[pick] += nu;
      received[pick] = 1;
      emptied[i] = 1;
      src_out[k] = s[i];
      dst_out[k] = s[pick];
      ++k;
    }
    *num_pairs = k;
  } catch (...) {
    return LAMINAR_ERR_INVALID_ARG;
  }
  return LAMINAR_OK;
}

laminar_status laminar_migration_pairs(const int32_t* src_table,
                                       const int32_t* lens, int32_t n_traj,
                                       int32_t src_width,
                                       const int32_t* dst_free, int32_t n_free,
                                       int32_t* dst_table, int32_t dst_width,
                                       int32_t* pairs, int32_t capacity,
                                       int32_t* num_pairs, int32_t* free_used) {
  if (!num_pairs || !free_used || n_traj < 0 || src_width < 0 || n_free < 0 ||
      dst_width < 0 || capacity < 0)
    return LAMINAR_ERR_INVALID_ARG;
  *num_pairs = 0;
  *free_used = 0;
  if (n_traj == 0) return LAMINAR_OK;
  if (!src_table || !lens || !dst_table || (n_free > 0 && !dst_free) ||
      (capacity > 0 && !pairs))
    return LAMINAR_ERR_INVALID_ARG;
  try {
    std::unordered_map<int32_t, int32_t> moved;   // source page -> dest page
    int32_t k = 0, used = 0;
    for (int32_t t = 0; t < n_traj; ++t) {
      if (lens[t] < 0) return LAMINAR_ERR_INVALID_ARG;
      const int64_t blocks = (int64_t(lens[t]) + 15) / 16;
      if (blocks > src_width || blocks > dst_width) return LAMINAR_ERR_INVALID_ARG;
      const int32_t* row = src_table + size_t(t) * src_width;
      int32_t* out = dst_table + size_t(t) * dst_width;
      for (int64_t j = 0; j < blocks; ++j) {
        const int32_t sp = row[j];
        if (sp < 0) return LAMINAR_ERR_INVALID_ARG;
        auto it = moved.find(sp);
        if (it == moved.end()) {
          if (used >= n_free || k >= capacity) return LAMINAR_ERR_INVALID_ARG;
          const int32_t dp = dst_free[used++];
          it = moved.emplace(sp, dp).first;
          pairs[2 * k] = sp;
          pairs[2 * k + 1] = dp;
          ++k;
        }
        out[j] = it->second;
      }
      for (int64_t j = blocks; j < dst_width; ++j) out[j] = -1;
    }
    *num_pairs = k;
    *free_used = used;
  } catch (...) {
    return LAMINAR_ERR_INVALID_ARG;
  }
  return LAMINAR_OK;
}


laminar_status laminar_roofline_batch_bound(const laminar_model_shape* m,
                                            uint64_t peak_flops,
                                            uint64_t peak_bw, int32_t* bound) {
  if (!bound || !shape_ok(m) || peak_flops == 0 || peak_bw == 0)
    return LAMINAR_ERR_INVALID_ARG;
  // sum N K and sum (K + N) over the projections
  __int128 nk = 0, kn = 0;
  for_each_projection(m, [&](int64_t k, int64_t n) {
    nk += __int128(k) * n;
    kn += k + n;
  });
  // compute-bound at M  <=>  M (2 nk BW - ab kn F) >= wb nk F
  const __int128 F = peak_flops, BW = peak_bw;
  const __int128 den = 2 * nk * BW - __int128(m->act_bytes) * kn * F;
  if (den <= 0) {
    *bound = 0;
    return LAMINAR_OK;
  }
  const __int128 num = __int128(m->weight_bytes) * nk * F;
  __int128 b = (num + den - 1) / den;
  if (b < 1) b = 1;
  *bound = b > INT32_MAX ? INT32_MAX : int32_t(b);
  return LAMINAR_OK;
}

laminar_status laminar_roofline_step_seconds(const laminar_model_shape* m,
                                             int64_t batch, int64_t context,
                                             uint64_t peak_flops,
                                             uint64_t peak_bw, double* seconds) {
  if (!seconds || !shape_ok(m) || peak_flops == 0 || peak_bw == 0 ||
      batch < 0 || context < 0)
    return LAMINAR_ERR_INVALID_ARG;
  const long double F = peak_flops, BW = peak_bw, M = batch;
  long double t = 0;
  for_each_projection(m, [&](int64_t k, int64_t n) {
    const long double flops = 2 * M * k * n;
    const long double bytes = (long double)(m->weight_bytes) * k * n +
                              (long double)(m->act_bytes) * M * (k + n);
    t += std::max(flops / F, bytes / BW);
  });
  const long double att_f = 4 * M * context * m->q_heads * m->head_dim;
  const long double att_b = (long double)(m->kv_bytes) * 2 * m->kv_heads *
                            m->head_dim * M * (context + 1);
  t += m->layers * std::max(att_f / F, att_b / BW);
  *seconds = double(t);
  return LAMINAR_OK;
}

}  // extern "C"
