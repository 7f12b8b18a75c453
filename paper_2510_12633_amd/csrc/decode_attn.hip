// Paged grouped-query decode attention for MI355X (gfx950, CDNA4).
//
// Rollout decoding is memory-bound (§2.4 of the paper) and its KV-cache reads
// dominate each decode step (§5.2), so the kernels below are organised around
// streaming 16-token KV pages from HBM once:
//
//  * decode_items: one workgroup per work item (trajectory, kv-head, page
//    range) of the host plan. Each wavefront takes pairs of pages in turn
//    and keeps the next pair's loads in flight while it computes the current
//    one. Per pair it forms the scores of all g query heads of the GQA group
//    with bf16 matrix-core products (v_mfma_f32_16x16x32_bf16: 16 tokens x
//    16 head slots, head_dim as the reduction), updates an online softmax in
//    fp32, and accumulates P*V on the matrix cores with P split into a bf16
//    high part and a bf16 low part, so P keeps about 16 bits of precision.
//    The page layouts put every operand fragment in 16-byte runs, so no LDS
//    staging or lane shuffles are needed; LDS is only used to combine the
//    wavefronts of one item. A cascade item (trajectories sharing a prompt
//    prefix) instead gives each wavefront the rows of 16/g members and lets
//    every wavefront walk all shared pages, so the pages are read from HBM
//    once for all members (the other wavefronts hit L2); each row is masked
//    at its own member's length.
//  * decode_merge_rows / decode_merge_heads: log-sum-exp merge of the
//    partial (out, lse) records of trajectories whose pages were split over
//    several items (or whose shared prefix was decoded by a cascade item);
//    one workgroup per record when records have few slots, one per
//    (record, head) with the slots reduced in parallel otherwise.
//
// The C-ABI entry points that validate a call and launch these kernels are
// in attn_entry.hip; this file holds the kernels and their launchers only.

#include <hip/hip_runtime.h>

#include <cmath>
#include <cstdint>
#include <cstring>
#include <mutex>

#include "attn_internal.h"
#include "laminar_decode_attn.h"
#include "plan_internal.h"

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef short s16x4 __attribute__((ext_vector_type(4)));

constexpr float kLog2e = 1.4426950408889634f;
// Mean partial slots per merge record up to which a workgroup per record
// merges faster than a workgroup per (record, head): measured 7 against
// 9 us on the agentic mix (2.2 slots per record) and 11 against 7 us on
// post-repack (23 slots).
constexpr int kRowsMergeMaxMeanSlots = 4;
constexpr double kLn2d = 0.6931471805599453;

struct DecodeArgs {
  const uint16_t* q;
  int64_t q_stride;       // elements between trajectories' query rows
  const uint8_t* k_pages;
  const uint8_t* v_pages;
  const float* k_scale;
  const float* v_scale;
  const int32_t* block_table;
  const int32_t* seq_lens;
  float* out;
  float* lse;
  float* o_part;
  float* lse_part;
  const int4* items;
  const int4* merges;
  int* tail_counter;      // dynamic tail: next tail item to hand out
  int32_t num_main, num_tail;
  const int4* cunits;     // cascade unit headers
  const int2* cmembers;   // cascade member records
  int32_t hq, hkv, group, max_blocks, num_pages;
  float scale_log2;  // softmax_scale * log2(e)
  float scale;       // softmax_scale
};

// Fragment geometry for one (page, kv-head) tile of 16 tokens x D dims.
template <int D, bool FP8>
struct Geo {
  static constexpr int KK = D / 32;             // QK^T matrix-core steps
  static constexpr int NT = D / 16;             // 16-dim tiles of P*V
  static constexpr int EB = FP8 ? 1 : 2;        // bytes per element
  static constexpr int TILE = 16 * D * EB;      // bytes per tile
  static constexpr int KL = 8 * KK * EB / 16;   // 16-byte K loads per lane
  static constexpr int VL = 4 * NT * EB / 16;   // 16-byte V loads per lane
  static constexpr int DPL = 4 / EB;            // dims per 16-byte V load
  // Dim of row m of P*V tile n. Load j of a lane in row m covers dims
  // j*16*DPL + m*DPL .. +DPL-1, so the 16 lanes of a group read one
  // contiguous 256-byte run per load; tile n is element n % DPL of load
  // n / DPL.
  static constexpr int vdim(int n, int m) {
    return (n / DPL) * 16 * DPL + m * DPL + n % DPL;
  }
};

template <int D, bool FP8>
struct PairRegs {
  using G = Geo<D, FP8>;
  u32x4 ka[G::KL], kb[G::KL];
  u32x4 va[G::VL], vb[G::VL];
  int nva, nvb;          // valid tokens in page A / B (0..16)
  int base;              // token index of slot 0 of page A
  float ksa, ksb, vsa, vsb;
};

__device__ __forceinline__ uint32_t pack_bf16(float lo, float hi) {
  bf16x2 v;
  v[0] = (__bf16)lo;     // round to nearest even (v_cvt_pk_bf16_f32)
  v[1] = (__bf16)hi;
  return __builtin_bit_cast(uint32_t, v);
}

// Two OCP e4m3fn codes (bytes 0,1 or, with HIGH, 2,3 of w) to a packed bf16
// pair; exact.
template <bool HIGH>
__device__ __forceinline__ uint32_t fp8x2_to_bf16x2(uint32_t w) {
  return __builtin_bit_cast(
      uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(w, 1.0f, HIGH));
}

__device__ __forceinline__ float bf16_lo_f(uint32_t w) {
  return __uint_as_float(w << 16);
}
__device__ __forceinline__ float bf16_hi_f(uint32_t w) {
  return __uint_as_float(w & 0xFFFF0000u);
}

__device__ __forceinline__ u32x4 u4(uint32_t a, uint32_t b, uint32_t c,
                                    uint32_t d) {
  u32x4 r;
  r[0] = a; r[1] = b; r[2] = c; r[3] = d;
  return r;
}

__device__ __forceinline__ s16x4 s4(uint32_t a, uint32_t b) {
  u32x2 r;
  r[0] = a; r[1] = b;
  return __builtin_bit_cast(s16x4, r);
}

__device__ __forceinline__ uint32_t word(const u32x4* v, int k) {
  return v[k >> 2][k & 3];
}

// A-operand fragment of K for matrix-core step kk: lane (token t = lane%16,
// group gq = lane/16) holds dims (gq*KK + kk)*8 .. +7 of token t.
template <int D, bool FP8>
__device__ __forceinline__ bf16x8 k_frag(const u32x4 (&k)[Geo<D, FP8>::KL],
                                         int kk) {
  if constexpr (!FP8) {
    return __builtin_bit_cast(bf16x8, k[kk]);
  } else {
    const u32x4 src = k[kk >> 1];
    const uint32_t w0 = src[(kk & 1) * 2], w1 = src[(kk & 1) * 2 + 1];
    return __builtin_bit_cast(
        bf16x8, u4(fp8x2_to_bf16x2<false>(w0), fp8x2_to_bf16x2<true>(w0),
                   fp8x2_to_bf16x2<false>(w1), fp8x2_to_bf16x2<true>(w1)));
  }
}

// A-operand fragment of V^T for dim tile n: lane (row m = lane%16, group gq)
// holds dim Geo::vdim(n, m) of tokens 4gq..4gq+3 of page A (items 0-3) and
// of page B (items 4-7).
template <int D, bool FP8>
__device__ __forceinline__ bf16x8 v_frag(const u32x4 (&va)[Geo<D, FP8>::VL],
                                         const u32x4 (&vb)[Geo<D, FP8>::VL],
                                         int n) {
  if constexpr (!FP8) {
    return __builtin_bit_cast(
        bf16x8, u4(word(va, 2 * n), word(va, 2 * n + 1), word(vb, 2 * n),
                   word(vb, 2 * n + 1)));
  } else {
    const uint32_t wa = word(va, n), wb = word(vb, n);
    return __builtin_bit_cast(
        bf16x8, u4(fp8x2_to_bf16x2<false>(wa), fp8x2_to_bf16x2<true>(wa),
                   fp8x2_to_bf16x2<false>(wb), fp8x2_to_bf16x2<true>(wb)));
  }
}

// Zero the V elements of tokens at or beyond `nv` held by this lane
// (tokens 4gq..4gq+3 of the page), so that P = 0 never meets NaN poison.
template <int D, bool FP8>
__device__ __forceinline__ void zero_tail_v(u32x4* v, int nv, int gq) {
  const int t0 = 4 * gq;
  if constexpr (!FP8) {
    const uint32_t m0 = (t0 + 0 < nv ? 0x0000FFFFu : 0u) |
                        (t0 + 1 < nv ? 0xFFFF0000u : 0u);
    const uint32_t m1 = (t0 + 2 < nv ? 0x0000FFFFu : 0u) |
                        (t0 + 3 < nv ? 0xFFFF0000u : 0u);
#pragma unroll
    for (int j = 0; j < Geo<D, FP8>::VL; ++j) {
      v[j][0] &= m0; v[j][1] &= m1; v[j][2] &= m0; v[j][3] &= m1;
    }
  } else {
    const uint32_t m = (t0 + 0 < nv ? 0x000000FFu : 0u) |
                       (t0 + 1 < nv ? 0x0000FF00u : 0u) |
                       (t0 + 2 < nv ? 0x00FF0000u : 0u) |
                       (t0 + 3 < nv ? 0xFF000000u : 0u);
#pragma unroll
    for (int j = 0; j < Geo<D, FP8>::VL; ++j) {
      v[j][0] &= m; v[j][1] &= m; v[j][2] &= m; v[j][3] &= m;
    }
  }
}

// Wave-uniform description of one work item.
struct ItemCtx {
  int b, kvh, len, p0, npages, slot;
};

__device__ __forceinline__ ItemCtx item_ctx(const DecodeArgs& a, int unit,
                                            int p0, int p1, int slot) {
  ItemCtx c;
  c.b = unit / a.hkv;
  c.kvh = unit - c.b * a.hkv;
  c.len = a.seq_lens[c.b];
  c.p0 = p0;
  c.npages = max(min(p1, (c.len + 15) >> 4) - c.p0, 0);
  c.slot = slot;
  return c;
}

// Query fragment (B operand of QK^T): lane holds the row of head slot r16
// (query head h of trajectory b when ok, zero otherwise), dims
// (gq*KK + kk)*8 .. +7 for each step kk.
template <int D, bool FP8>
__device__ __forceinline__ void load_q(const DecodeArgs& a, int b, int h,
                                       bool ok, int gq,
                                       bf16x8 (&qf)[Geo<D, FP8>::KK]) {
  using G = Geo<D, FP8>;
  const u32x4* qp = reinterpret_cast<const u32x4*>(
      a.q + size_t(ok ? b : 0) * a.q_stride + size_t(ok ? h : 0) * D) +
      gq * G::KK;
#pragma unroll
  for (int kk = 0; kk < G::KK; ++kk) {
    const u32x4 v = ok ? qp[kk] : u4(0, 0, 0, 0);
    qf[kk] = __builtin_bit_cast(bf16x8, v);
  }
}

// Issue the loads of pages ja and ja+1 of the item (ja even). The two
// block-table entries are read through the scalar cache (the index is
// wave-uniform), and each page is read through a buffer resource whose size
// is the tile for a valid page and zero otherwise: pages past the item
// (including the whole pair after the last one, issued unconditionally),
// table entries outside the pool and the second page of an odd tail read
// zeros without touching memory. No load is conditional, so the compiler
// counts the loads in flight exactly and the next pair's loads overlap the
// current pair's arithmetic.
typedef const __attribute__((address_space(4))) int32_t* ConstI32;
typedef const __attribute__((address_space(4))) float* ConstF32;
constexpr int kBufFlags = 0x00020000;

template <int D, bool FP8>
__device__ __forceinline__ void issue_pair(const DecodeArgs& a,
                                           const ItemCtx& c, int ja,
                                           int koff, int voff,
                                           PairRegs<D, FP8>& pr) {
  using G = Geo<D, FP8>;
  const ConstI32 row =
      (ConstI32)(a.block_table + size_t(c.b) * a.max_blocks + c.p0);
  const int last = max(c.npages - 1, 0);
  int ppa = row[min(ja, last)];
  int ppb = row[min(ja + 1, last)];
  const int base_tok = (c.p0 + ja) * 16;
  int nva = ja < c.npages ? min(16, c.len - base_tok) : 0;
  int nvb = ja + 1 < c.npages ? min(16, c.len - base_tok - 16) : 0;
  if (ppa < 0 || ppa >= a.num_pages) { ppa = 0; nva = 0; }
  if (ppb < 0 || ppb >= a.num_pages) { ppb = 0; nvb = 0; }
  pr.nva = nva;
  pr.nvb = nvb;
  pr.base = base_tok;
  const size_t page_stride = size_t(a.hkv) * G::TILE;
  uint8_t* kbase = const_cast<uint8_t*>(a.k_pages) + size_t(c.kvh) * G::TILE;
  uint8_t* vbase = const_cast<uint8_t*>(a.v_pages) + size_t(c.kvh) * G::TILE;
  const __amdgpu_buffer_rsrc_t kra = __builtin_amdgcn_make_buffer_rsrc(
      kbase + size_t(ppa) * page_stride, 0, nva > 0 ? G::TILE : 0, kBufFlags);
  const __amdgpu_buffer_rsrc_t krb = __builtin_amdgcn_make_buffer_rsrc(
      kbase + size_t(ppb) * page_stride, 0, nvb > 0 ? G::TILE : 0, kBufFlags);
  const __amdgpu_buffer_rsrc_t vra = __builtin_amdgcn_make_buffer_rsrc(
      vbase + size_t(ppa) * page_stride, 0, nva > 0 ? G::TILE : 0, kBufFlags);
  const __amdgpu_buffer_rsrc_t vrb = __builtin_amdgcn_make_buffer_rsrc(
      vbase + size_t(ppb) * page_stride, 0, nvb > 0 ? G::TILE : 0, kBufFlags);
  // KV pages are streamed once per call: non-temporal loads keep them from
  // displacing reusable lines in L2 and the Infinity Cache.
#pragma unroll
  for (int j = 0; j < G::KL; ++j)
    pr.ka[j] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(
        kra, (koff + j * 16) * 16, 0, 2));
#pragma unroll
  for (int j = 0; j < G::KL; ++j)
    pr.kb[j] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(
        krb, (koff + j * 16) * 16, 0, 2));
#pragma unroll
  for (int j = 0; j < G::VL; ++j)
    pr.va[j] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(
        vra, (voff + j * 16) * 16, 0, 2));
#pragma unroll
  for (int j = 0; j < G::VL; ++j)
    pr.vb[j] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(
        vrb, (voff + j * 16) * 16, 0, 2));
  if constexpr (FP8) {
    const ConstF32 ks = (ConstF32)(a.k_scale);
    const ConstF32 vs = (ConstF32)(a.v_scale);
    pr.ksa = ks[size_t(ppa) * a.hkv + c.kvh];
    pr.ksb = ks[size_t(ppb) * a.hkv + c.kvh];
    pr.vsa = vs[size_t(ppa) * a.hkv + c.kvh];
    pr.vsb = vs[size_t(ppb) * a.hkv + c.kvh];
  }
}

// Running softmax state of the wave for the g heads of one item: lane
// (head r16, group gq) holds the running max of head r16 (identical across
// groups) as mc = max(score) * scale * log2(e) rounded once, its share of
// the denominator sum(exp2(score * scale * log2(e) - mc)), and output rows
// 4gq..4gq+3 of every 16-dim tile. Keeping the rounded mc itself makes the
// rescale factor exp2(mc_old - mc_new) exactly 1 while the max is unchanged
// (no drift over thousands of pages) and lets lse = mc * ln 2 + ln(l) use
// the very offset the exponentials used.
template <int D>
struct Acc {
  f32x4 o[D / 16];
  float m;     // mc, in log2 units; -inf before the first valid token
  float l;
  __device__ __forceinline__ void reset() {
#pragma unroll
    for (int n = 0; n < D / 16; ++n) o[n] = f32x4{0.f, 0.f, 0.f, 0.f};
    m = -INFINITY;
    l = 0.f;
  }
};

template <int D, bool FP8>
__device__ __forceinline__ void compute_pair(const DecodeArgs& a,
                                             const bf16x8 (&qf)[Geo<D, FP8>::KK],
                                             PairRegs<D, FP8>& pr, Acc<D>& st,
                                             int gq, bool rows,
                                             const int* row_len_lds) {
  using G = Geo<D, FP8>;
  // Scores S^T[token][head] of both pages: lane holds head r16, tokens
  // 4gq..4gq+3 of page A (sa) and of page B (sb).
  f32x4 sa = {0.f, 0.f, 0.f, 0.f}, sb = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int kk = 0; kk < G::KK; ++kk) {
    sa = __builtin_amdgcn_mfma_f32_16x16x32_bf16(k_frag<D, FP8>(pr.ka, kk),
                                                 qf[kk], sa, 0, 0, 0);
    sb = __builtin_amdgcn_mfma_f32_16x16x32_bf16(k_frag<D, FP8>(pr.kb, kk),
                                                 qf[kk], sb, 0, 0, 0);
  }
  if constexpr (FP8) {
    sa *= pr.ksa;
    sb *= pr.ksb;
  }
  // Slots past the page's valid tokens score -inf, and so do slots past
  // the length of this lane's row when rows belong to different members
  // (`rows`, a cascade item; the lengths sit in LDS, not in registers).
  if (rows || pr.nva < 16 || pr.nvb < 16) {    // uniform
    int la = pr.nva, lb = pr.nvb;
    if (rows) {
      // this lane's row: entry (wavefront, head slot) of the LDS table
      const int rl = __atomic_load_n(&row_len_lds[(threadIdx.x >> 6) * 16 +
                                                  (threadIdx.x & 15)],
                                     __ATOMIC_RELAXED) - pr.base;
      la = min(la, rl);
      lb = min(lb, rl - 16);
    }
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      sa[r] = (4 * gq + r < la) ? sa[r] : -INFINITY;
      sb[r] = (4 * gq + r < lb) ? sb[r] : -INFINITY;
    }
    if (pr.nva < 16 || pr.nvb < 16) {
      zero_tail_v<D, FP8>(pr.va, pr.nva, gq);
      zero_tail_v<D, FP8>(pr.vb, pr.nvb, gq);
    }
  }
  float mx = fmaxf(fmaxf(fmaxf(sa[0], sa[1]), fmaxf(sa[2], sa[3])),
                   fmaxf(fmaxf(sb[0], sb[1]), fmaxf(sb[2], sb[3])));
  mx = fmaxf(mx, __shfl_xor(mx, 16));
  mx = fmaxf(mx, __shfl_xor(mx, 32));
  const float mc_new = fmaxf(st.m, mx * a.scale_log2);   // -inf stays -inf
  const float alpha = (st.m == -INFINITY)
                          ? 0.f
                          : __builtin_amdgcn_exp2f(st.m - mc_new);
  const float mc = (mc_new == -INFINITY) ? 0.f : mc_new;
  st.m = mc_new;
  float pa[4], pb[4];
#pragma unroll
  for (int r = 0; r < 4; ++r) {
    pa[r] = __builtin_amdgcn_exp2f(fmaf(sa[r], a.scale_log2, -mc));
    pb[r] = __builtin_amdgcn_exp2f(fmaf(sb[r], a.scale_log2, -mc));
  }
  st.l = fmaf(st.l, alpha, ((pa[0] + pa[1]) + (pa[2] + pa[3])) +
                               ((pb[0] + pb[1]) + (pb[2] + pb[3])));
#pragma unroll
  for (int n = 0; n < G::NT; ++n) st.o[n] *= alpha;
  if constexpr (FP8) {
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      pa[r] *= pr.vsa;
      pb[r] *= pr.vsb;
    }
  }
  // P^T as B operand: lane holds head r16, slots 8gq+e = token 4gq+e of
  // page A (e < 4) and of page B (e >= 4); P = hi + lo in bf16.
  const uint32_t h0 = pack_bf16(pa[0], pa[1]), h1 = pack_bf16(pa[2], pa[3]);
  const uint32_t h2 = pack_bf16(pb[0], pb[1]), h3 = pack_bf16(pb[2], pb[3]);
  const uint32_t l0 = pack_bf16(pa[0] - bf16_lo_f(h0), pa[1] - bf16_hi_f(h0));
  const uint32_t l1 = pack_bf16(pa[2] - bf16_lo_f(h1), pa[3] - bf16_hi_f(h1));
  const uint32_t l2 = pack_bf16(pb[0] - bf16_lo_f(h2), pb[1] - bf16_hi_f(h2));
  const uint32_t l3 = pack_bf16(pb[2] - bf16_lo_f(h3), pb[3] - bf16_hi_f(h3));
  if constexpr (!FP8) {
    // bf16 V: one 16x16x16 product per page; its A operand (tile row r16,
    // tokens 4gq..4gq+3) is two of the loaded registers.
    const s16x4 pha = s4(h0, h1), pla = s4(l0, l1);
    const s16x4 phb = s4(h2, h3), plb = s4(l2, l3);
#pragma unroll
    for (int n = 0; n < G::NT; ++n) {
      const s16x4 vta = s4(word(pr.va, 2 * n), word(pr.va, 2 * n + 1));
      const s16x4 vtb = s4(word(pr.vb, 2 * n), word(pr.vb, 2 * n + 1));
      st.o[n] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(vta, pha, st.o[n], 0, 0, 0);
      st.o[n] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(vta, pla, st.o[n], 0, 0, 0);
      st.o[n] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(vtb, phb, st.o[n], 0, 0, 0);
      st.o[n] = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(vtb, plb, st.o[n], 0, 0, 0);
    }
  } else {
    // fp8 V: the converted registers form one 16x16x32 operand per tile,
    // tokens of page A in items 0-3 and of page B in items 4-7.
    const bf16x8 phi = __builtin_bit_cast(bf16x8, u4(h0, h1, h2, h3));
    const bf16x8 plo = __builtin_bit_cast(bf16x8, u4(l0, l1, l2, l3));
#pragma unroll
    for (int n = 0; n < G::NT; ++n) {
      const bf16x8 vt = v_frag<D, FP8>(pr.va, pr.vb, n);
      st.o[n] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vt, phi, st.o[n], 0, 0, 0);
      st.o[n] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vt, plo, st.o[n], 0, 0, 0);
    }
  }
}

// Write one query row's result (out or partial row `dst`, lse at `lse_dst`)
// from lane (head slot, group gq). st.l must already hold the full
// denominator of the row.
template <int D, bool FP8>
__device__ __forceinline__ void write_row(float* dst, float* lse_dst,
                                          const Acc<D>& st, int gq) {
  using G = Geo<D, FP8>;
  const bool empty = !(st.l > 0.f);
  const float inv = empty ? 0.f : 1.0f / st.l;
  const float lse_v =
      empty ? -INFINITY : float(double(st.m) * kLn2d + log(double(st.l)));
  // Row 4gq + r of tile n is dim vdim(n, 4gq + r): for each load j the lane
  // holds 4*DPL contiguous dims starting at j*16*DPL + 4gq*DPL, ordered
  // (r, e) with n = j*DPL + e.
#pragma unroll
  for (int j = 0; j < G::NT / G::DPL; ++j) {
    float vals[4 * G::DPL];
#pragma unroll
    for (int r = 0; r < 4; ++r)
#pragma unroll
      for (int e = 0; e < G::DPL; ++e)
        vals[r * G::DPL + e] = st.o[j * G::DPL + e][r] * inv;
    float4* run = reinterpret_cast<float4*>(dst + G::vdim(j * G::DPL, 4 * gq));
#pragma unroll
    for (int k = 0; k < G::DPL; ++k)
      run[k] = make_float4(vals[4 * k], vals[4 * k + 1], vals[4 * k + 2],
                           vals[4 * k + 3]);
  }
  if (gq == 0) *lse_dst = lse_v;
}

// Result of an ordinary item: out/lse directly when the trajectory was not
// split, else the partial record of its slot.
template <int D, bool FP8>
__device__ __forceinline__ void write_item(const DecodeArgs& a,
                                           const ItemCtx& c, const Acc<D>& st,
                                           int r16, int gq) {
  if (r16 >= a.group) return;
  const int h = c.kvh * a.group + r16;
  if (c.slot < 0)
    write_row<D, FP8>(a.out + (size_t(c.b) * a.hq + h) * D,
                      a.lse + size_t(c.b) * a.hq + h, st, gq);
  else
    write_row<D, FP8>(a.o_part + (size_t(c.slot) * a.group + r16) * D,
                      a.lse_part + size_t(c.slot) * a.group + r16, st, gq);
}

// One workgroup per work item (trajectory, kv-head, page range), in the
// plan's longest-first order; the hardware dispatcher hands items to CUs as
// workgroups finish, and the plan's smallest items (the dynamic tail) go to
// whichever workgroup starts next. The WAVES wavefronts share the item's page pairs (wave
// w takes pairs w, w+WAVES, ...), each keeping the next pair's loads in
// flight while it computes the current one; the waves are combined through
// LDS at the end and wave 0 writes the result.
template <int D, bool FP8, int WAVES, bool CASCADE>
__global__ void __launch_bounds__(64 * WAVES)
__attribute__((amdgpu_waves_per_eu(2)))
decode_items(const DecodeArgs a) {
  using G = Geo<D, FP8>;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  int k = blockIdx.x;
  if (!CASCADE && k >= a.num_main) {
    // Dynamic tail: this workgroup takes the next tail item (longest
    // first) when the hardware starts it, on whichever XCD has room. Every
    // tail workgroup pulls once; the pull that gets the last index resets
    // the counter for the next launch.
    __shared__ int s_idx;
    if (threadIdx.x == 0) {
      const int t = __hip_atomic_fetch_add(a.tail_counter, 1, __ATOMIC_RELAXED,
                                           __HIP_MEMORY_SCOPE_AGENT);
      if (t == a.num_tail - 1)
        __hip_atomic_store(a.tail_counter, 0, __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
      s_idx = t;
    }
    __syncthreads();
    if (s_idx >= a.num_tail) return;     // not expected; keeps k in range
    k = a.num_main + s_idx;
  }
  {
    using G = Geo<D, FP8>;
    const int r16 = lane & 15, gq = lane >> 4;
    const int koff = gq * G::KL * 16 + r16;                    // u32x4 units
    const int voff = gq * D * G::EB / 4 + r16;                  // u32x4 units
    const int4 it = a.items[k];
    // uniform; plans without cascade items run the CASCADE = false
    // instantiation, which carries none of the cascade code
    const bool cascade = CASCADE && it.x < 0;
    ItemCtx c;
    int4 cu = make_int4(0, 0, 0, 0);     // cascade unit header
    // Tokens a cascade row may attend to (its member's length), kept in LDS
    // rather than a register through the page loop; ordinary rows use c.len.
    __shared__ int sm_row_len[WAVES * 16];
    // page pairs of this wavefront: jp0, jp0 + stride, ...
    int jp0 = wave, stride = WAVES;
    bf16x8 qf[G::KK];
    if (!cascade) {
      c = item_ctx(a, it.x, it.y, it.z, it.w);
      load_q<D, FP8>(a, c.b, c.kvh * a.group + r16, r16 < a.group, gq, qf);
    } else {
      // Cascade item: shared pages read through the longest member's table
      // row; wavefront w holds the rows of members w*mw .. w*mw + mw - 1
      // (mw = 16 / g), head r16 % g of member w*mw + r16 / g in lane r16.
      cu = a.cunits[-it.x - 1];
      c = item_ctx(a, cu.x * a.hkv + cu.w, it.y, it.z, it.w);
      const int mw = 16 / a.group;
      if (wave * mw >= cu.y) return;          // no members for this wave
      const int mi = wave * mw + r16 / a.group;
      const bool ok = r16 < mw * a.group && mi < cu.y;
      const int rb = ok ? a.cmembers[cu.z + mi].x : 0;
      if (gq == 0) sm_row_len[wave * 16 + r16] = ok ? a.seq_lens[rb] : 0;
      jp0 = 0;
      stride = 1;
      load_q<D, FP8>(a, rb, c.kvh * a.group + r16 % a.group, ok, gq, qf);
    }
    const int npairs = (c.npages + 1) >> 1;
    Acc<D> st;
    st.reset();

    PairRegs<D, FP8> buf0, buf1;
    int jp = jp0;
    issue_pair<D, FP8>(a, c, 2 * jp, koff, voff, buf0);
    while (jp < npairs) {
      int jn = jp + stride;
      issue_pair<D, FP8>(a, c, 2 * jn, koff, voff, buf1);
      __builtin_amdgcn_sched_barrier(0);   // next pair's loads go out first
      compute_pair<D, FP8>(a, qf, buf0, st, gq, cascade, sm_row_len);
      jp = jn;
      if (jp >= npairs) break;
      jn = jp + stride;
      issue_pair<D, FP8>(a, c, 2 * jn, koff, voff, buf0);
      __builtin_amdgcn_sched_barrier(0);
      compute_pair<D, FP8>(a, qf, buf1, st, gq, cascade, sm_row_len);
      jp = jn;
    }

    // Full softmax denominator of head r16 over this wave's pages.
    st.l += __shfl_xor(st.l, 16);
    st.l += __shfl_xor(st.l, 32);

    if (cascade) {                 // each wavefront owns its rows: no combine
      const int mw = 16 / a.group;
      const int mi = wave * mw + r16 / a.group;
      if (r16 < mw * a.group && mi < cu.y) {
        const int slot = a.cmembers[cu.z + mi].y + c.slot;
        const int i = r16 % a.group;
        write_row<D, FP8>(a.o_part + (size_t(slot) * a.group + i) * D,
                          a.lse_part + size_t(slot) * a.group + i, st, gq);
      }
      return;
    }

    if constexpr (WAVES > 1) {
      __shared__ float sm_m[WAVES][16];
      __shared__ float sm_l[WAVES][16];
      __shared__ float sm_acc[WAVES - 1][G::NT * 4][64];
      if (wave > 0) {
        if (gq == 0) {
          sm_m[wave][r16] = st.m;
          sm_l[wave][r16] = st.l;
        }
#pragma unroll
        for (int n = 0; n < G::NT; ++n)
#pragma unroll
          for (int r = 0; r < 4; ++r)
            sm_acc[wave - 1][n * 4 + r][lane] = st.o[n][r];
      }
      __syncthreads();
      if (wave == 0) {
        float m_all = st.m;
#pragma unroll
        for (int w = 1; w < WAVES; ++w) m_all = fmaxf(m_all, sm_m[w][r16]);
        const float mref = (m_all == -INFINITY) ? 0.f : m_all;
        const float f0 = __builtin_amdgcn_exp2f(st.m - mref);   // 0 for -inf
        st.l *= f0;
#pragma unroll
        for (int n = 0; n < G::NT; ++n) st.o[n] *= f0;
#pragma unroll
        for (int w = 1; w < WAVES; ++w) {
          const float fw = __builtin_amdgcn_exp2f(sm_m[w][r16] - mref);
          st.l = fmaf(sm_l[w][r16], fw, st.l);
#pragma unroll
          for (int n = 0; n < G::NT; ++n)
#pragma unroll
            for (int r = 0; r < 4; ++r)
              st.o[n][r] = fmaf(sm_acc[w - 1][n * 4 + r][lane], fw, st.o[n][r]);
        }
        st.m = m_all;
      }
      __syncthreads();          // LDS is reused by the next item
      if (wave == 0) write_item<D, FP8>(a, c, st, r16, gq);
    } else {
      write_item<D, FP8>(a, c, st, r16, gq);
    }
  }
}

// Block-wide reductions for 256 threads.
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

// Merge for records with few slots (cascade members: the shared prefix's
// partial and one or two of their own): one workgroup per merge record;
// thread (head i, column c) merges the n partial rows of head i for dims
// 4c..4c+3. The lse values of a head are read by its D/4 threads together
// (one cache line), and every load's address is known up front, so the
// loops keep many loads in flight.
template <int D>
__global__ void __launch_bounds__(256) decode_merge_rows(const DecodeArgs a) {
  constexpr int C = D / 4;          // float4 columns per row
  const int4 mg = a.merges[blockIdx.x];
  const int unit = mg.x, slot0 = mg.y, n = mg.z;
  const int b = unit / a.hkv;
  const int kvh = unit - b * a.hkv;
  for (int t = threadIdx.x; t < a.group * C; t += 256) {
    const int i = t / C, c = t - i * C;
    const float* lp = a.lse_part + size_t(slot0) * a.group + i;
    const float4* op =
        reinterpret_cast<const float4*>(a.o_part + (size_t(slot0) * a.group + i) * D) + c;
    const size_t ostride = size_t(a.group) * C;        // float4 per slot
    float mx = -INFINITY;
#pragma unroll 4
    for (int s = 0; s < n; ++s) mx = fmaxf(mx, lp[size_t(s) * a.group]);
    float sum = 0.f;
    float4 o = make_float4(0.f, 0.f, 0.f, 0.f);
    if (mx != -INFINITY) {
#pragma unroll 4
      for (int s = 0; s < n; ++s) {
        const float w = expf(lp[size_t(s) * a.group] - mx);   // 0 for -inf
        const float4 v = op[size_t(s) * ostride];
        sum += w;
        o.x = fmaf(w, v.x, o.x); o.y = fmaf(w, v.y, o.y);
        o.z = fmaf(w, v.z, o.z); o.w = fmaf(w, v.w, o.w);
      }
    }
    const int h = kvh * a.group + i;
    const float inv = mx == -INFINITY ? 0.f : 1.0f / sum;
    reinterpret_cast<float4*>(a.out + (size_t(b) * a.hq + h) * D)[c] =
        make_float4(o.x * inv, o.y * inv, o.z * inv, o.w * inv);
    if (c == 0) a.lse[size_t(b) * a.hq + h] = mx == -INFINITY ? -INFINITY
                                                              : mx + logf(sum);
  }
}

// Merge with the slots in parallel, for records with many slots: one
// workgroup per (merge record, head of the group); 256 / (D/4) partial rows
// are reduced side by side and combined through LDS.
template <int D>
__global__ void __launch_bounds__(256) decode_merge_heads(const DecodeArgs a) {
  constexpr int C = D / 4;          // threads per partial row (float4 each)
  constexpr int SPAR = 256 / C;     // partial rows reduced in parallel
  __shared__ float red[4];
  __shared__ float4 part[SPAR][C];
  const int tid = threadIdx.x;
  const int4 mg = a.merges[blockIdx.x];
  const int i = blockIdx.y;
  const int unit = mg.x, slot0 = mg.y, n = mg.z;
  const int b = unit / a.hkv;
  const int kvh = unit - b * a.hkv;
  const int h = kvh * a.group + i;
  const float* lp = a.lse_part + size_t(slot0) * a.group + i;

  float mx = -INFINITY;
  for (int s = tid; s < n; s += 256) mx = fmaxf(mx, lp[size_t(s) * a.group]);
  mx = wave_max(mx);
  if ((tid & 63) == 0) red[tid >> 6] = mx;
  __syncthreads();
  mx = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
  __syncthreads();
  float sum = 0.f;
  if (mx != -INFINITY)
    for (int s = tid; s < n; s += 256) sum += expf(lp[size_t(s) * a.group] - mx);
  sum = wave_sum(sum);
  if ((tid & 63) == 0) red[tid >> 6] = sum;
  __syncthreads();
  sum = (red[0] + red[1]) + (red[2] + red[3]);
  const float L = (mx == -INFINITY) ? -INFINITY : mx + logf(sum);

  const int c = tid % C, s0 = tid / C;
  float4 o = make_float4(0.f, 0.f, 0.f, 0.f);
  if (L != -INFINITY) {
    for (int s = s0; s < n; s += SPAR) {
      const float w = expf(lp[size_t(s) * a.group] - L);
      const float4 v = reinterpret_cast<const float4*>(
          a.o_part + (size_t(slot0 + s) * a.group + i) * D)[c];
      o.x = fmaf(w, v.x, o.x); o.y = fmaf(w, v.y, o.y);
      o.z = fmaf(w, v.z, o.z); o.w = fmaf(w, v.w, o.w);
    }
  }
  part[s0][c] = o;
  __syncthreads();
  if (s0 == 0) {
    for (int s = 1; s < SPAR; ++s) {
      const float4 v = part[s][c];
      o.x += v.x; o.y += v.y; o.z += v.z; o.w += v.w;
    }
    reinterpret_cast<float4*>(a.out + (size_t(b) * a.hq + h) * D)[c] = o;
    if (c == 0) a.lse[size_t(b) * a.hq + h] = L;
  }
}

template <int D, bool FP8, bool CASCADE>
hipError_t launch_items(const laminar_plan& p, const DecodeArgs& a,
                        hipStream_t stream) {
  const dim3 grid(p.num_items);
  switch (p.waves) {
    case 1:
      hipLaunchKernelGGL((decode_items<D, FP8, 1, CASCADE>), grid, dim3(64), 0,
                         stream, a);
      break;
    case 2:
      hipLaunchKernelGGL((decode_items<D, FP8, 2, CASCADE>), grid, dim3(128), 0,
                         stream, a);
      break;
    default:
      hipLaunchKernelGGL((decode_items<D, FP8, 4, CASCADE>), grid, dim3(256), 0,
                         stream, a);
      break;
  }
  return hipGetLastError();
}

template <int D, bool FP8>
hipError_t launch_partial(const laminar_plan& p, const DecodeArgs& a,
                          hipStream_t stream) {
  return p.num_cascade_units > 0 ? launch_items<D, FP8, true>(p, a, stream)
                                 : launch_items<D, FP8, false>(p, a, stream);
}

DecodeArgs make_args(const laminar_plan& p,
                     const laminar_detail::AttnCall& c) {
  DecodeArgs a;
  const laminar_attn_desc& d = p.desc;
  char* ws = static_cast<char*>(c.ws);
  a.q = static_cast<const uint16_t*>(c.q);
  a.q_stride = d.input_row_stride ? d.input_row_stride
                                  : int64_t(d.num_q_heads) * d.head_dim;
  a.k_pages = static_cast<const uint8_t*>(c.k_pages);
  a.v_pages = static_cast<const uint8_t*>(c.v_pages);
  a.k_scale = d.k_scale;
  a.v_scale = d.v_scale;
  a.block_table = c.block_table;
  a.seq_lens = c.seq_lens;
  a.out = c.out;
  a.lse = c.lse;
  a.items = reinterpret_cast<const int4*>(ws + p.off_items);
  a.merges = reinterpret_cast<const int4*>(ws + p.off_merges);
  a.tail_counter = reinterpret_cast<int*>(ws + p.off_tail);
  a.num_main = p.num_main;
  a.num_tail = p.num_items - p.num_main;
  a.cunits = reinterpret_cast<const int4*>(ws + p.off_cunits);
  a.cmembers = reinterpret_cast<const int2*>(ws + p.off_cmembers);
  a.lse_part = reinterpret_cast<float*>(ws + p.off_lse);
  a.o_part = reinterpret_cast<float*>(ws + p.off_o);
  a.hq = d.num_q_heads;
  a.hkv = d.num_kv_heads;
  a.group = p.group;
  a.max_blocks = d.max_blocks_per_seq;
  a.num_pages = d.num_pages;
  a.scale_log2 = d.softmax_scale * kLog2e;
  a.scale = d.softmax_scale;
  return a;
}

}  // namespace

namespace laminar_detail {

laminar_status enqueue_partial(const laminar_plan& p, const AttnCall& c,
                               hipStream_t stream) {
  if (p.num_items == 0) return LAMINAR_OK;
  const DecodeArgs a = make_args(p, c);
  const bool fp8 = p.desc.kv_dtype == LAMINAR_KV_FP8_E4M3FN;
  hipError_t e;
  if (p.desc.head_dim == 128)
    e = fp8 ? launch_partial<128, true>(p, a, stream)
            : launch_partial<128, false>(p, a, stream);
  else
    e = fp8 ? launch_partial<64, true>(p, a, stream)
            : launch_partial<64, false>(p, a, stream);
  return e == hipSuccess ? LAMINAR_OK : LAMINAR_ERR_HIP;
}

laminar_status enqueue_merge(const laminar_plan& p, const AttnCall& c,
                             hipStream_t stream) {
  if (p.num_merges == 0) return LAMINAR_OK;
  const DecodeArgs a = make_args(p, c);
  // Few slots per record: a workgroup per record; many: a workgroup per
  // (record, head) reducing slots in parallel.
  const bool rows = p.num_slots <= kRowsMergeMaxMeanSlots * p.num_merges;
  const dim3 grid = rows ? dim3(p.num_merges) : dim3(p.num_merges, p.group);
  if (p.desc.head_dim == 128) {
    if (rows)
      hipLaunchKernelGGL((decode_merge_rows<128>), grid, dim3(256), 0, stream, a);
    else
      hipLaunchKernelGGL((decode_merge_heads<128>), grid, dim3(256), 0, stream, a);
  } else {
    if (rows)
      hipLaunchKernelGGL((decode_merge_rows<64>), grid, dim3(256), 0, stream, a);
    else
      hipLaunchKernelGGL((decode_merge_heads<64>), grid, dim3(256), 0, stream, a);
  }
  return hipGetLastError() == hipSuccess ? LAMINAR_OK : LAMINAR_ERR_HIP;
}

}  // namespace laminar_detail
